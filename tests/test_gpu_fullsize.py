"""Full-size parity on the four large workloads, in the launch configuration
bench.py times (SharedStep defaults: fused replay, default n_seed).

The full fp64 oracle cannot run at these sizes, so the comparison uses
``oracle.sampled`` on chosen rows:
* query rows (first/last rows of groups and branches plus random rows) of two
  query heads: O, LSE, dQ;
* key rows near the end of branches (dK_R, dV_R) and, where affordable, near
  the end of a prompt (dK_P, dV_P: the Eq. 2 total over the prefill and every
  branch);
and an identity that holds at any size: for every group and KV head, the sum
of dV over all its keys (prompt and branches) equals the sum of dO over the
query rows and query heads that read them (each softmax row sums to one).
"""
import types

import numpy as np
import pytest
import torch

from oracle import sampled as S
from paper_2609_33133_amd import inputs as I
from paper_2609_33133_amd.api import GroupBatch
from paper_2609_33133_amd.group_attention import SharedStep, upload

from gpu_helpers import TOL_GRAD, TOL_LSE, TOL_O, log, rel

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

# largest (query rows x keys x query heads) spent on one prompt-key reference
PROMPT_KEY_BUDGET = 2.5e9


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _sample_rows(rng, starts_ends, n_random, total):
    rows = set()
    for a, b in starts_ends:
        rows.update((a, b - 1))
    rows.update(int(x) for x in rng.integers(0, total, size=n_random))
    return sorted(rows)


def _host(t):
    return t.float().cpu().numpy().astype(np.float64)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["balanced", "prompt", "response", "ragged", "gsweep64", "prompt_gqa7"])
def test_fullsize_sampled(name):
    log(f"[fullsize] {name}: generating inputs")
    gi = I.make_config(name)
    s = gi.shape
    b = GroupBatch.from_shape(s)
    x = upload(gi, "cuda")
    step = SharedStep(b, "cuda")
    log(f"[fullsize] {name}: running the hot path (n_seed={step.n_seed})")
    step.run(x)
    torch.cuda.synchronize()
    out = step.outputs()
    for k, v in out.items():
        assert torch.isfinite(v.float()).all(), k

    t = types.SimpleNamespace(cu_prompt=s.cu_prompt, cu_branch=s.cu_branch, cu_resp=s.cu_resp,
                              num_q_heads=s.num_q_heads, num_kv_heads=s.num_kv_heads, head_dim=s.head_dim,
                              **{n: getattr(gi, n) for n in ("q_p", "k_p", "v_p", "q_r", "k_r", "v_r", "do_p",
                                                             "do_r")})
    rng = np.random.default_rng(123)
    groups = list(range(min(3, s.num_groups)))
    p_rows = _sample_rows(rng, [(int(s.cu_prompt[g]), int(s.cu_prompt[g + 1])) for g in groups], 6, s.total_prompt)
    br = [0, s.num_branches - 1, int(rng.integers(0, s.num_branches))]
    r_rows = _sample_rows(rng, [(int(s.cu_resp[i]), int(s.cu_resp[i + 1])) for i in br], 6, s.total_resp)

    # ---- query rows
    for h in (0, s.num_q_heads - 1):
        for kind, rows, o, lse, dq in (("prompt", p_rows, "o_p", "lse_p", "dq_p"),
                                       ("resp", r_rows, "o_r", "lse_r", "dq_r")):
            ref = S.query_rows(t, kind, rows, h)
            idx = torch.tensor(rows, device="cuda")
            go = _host(out[o].index_select(0, idx)[:, h])
            gl = _host(out[lse][h].index_select(0, idx))
            gd = _host(out[dq].index_select(0, idx)[:, h])
            eo, el, ed = rel(go, ref["o"]), float(np.max(np.abs(gl - ref["lse"]))), rel(gd, ref["dq"])
            log(f"[fullsize] {name} {kind} rows head {h}: O {eo:.2e} LSE {el:.2e} dQ {ed:.2e}")
            assert eo <= TOL_O and el <= TOL_LSE and ed <= TOL_GRAD

    # ---- response keys near the end of branches
    for bi in br[:2]:
        r0, r1 = int(s.cu_resp[bi]), int(s.cu_resp[bi + 1])
        rows = sorted({max(r0, r1 - 1), max(r0, r1 - 37), max(r0, r1 - 200)})
        for kh in (0, s.num_kv_heads - 1):
            ref = S.key_rows(t, "resp", rows, kh)
            idx = torch.tensor(rows, device="cuda")
            gk = _host(out["dk_r"].index_select(0, idx)[:, kh])
            gv = _host(out["dv_r"].index_select(0, idx)[:, kh])
            ek, ev = rel(gk, ref["dk"]), rel(gv, ref["dv"])
            log(f"[fullsize] {name} branch {bi} keys kv {kh}: dK {ek:.2e} dV {ev:.2e}")
            assert ek <= TOL_GRAD and ev <= TOL_GRAD

    # ---- prompt keys near the end of the cheapest group (Eq. 2 total)
    gq = s.num_q_heads // s.num_kv_heads

    def cost(g):
        P = s.prompt_lens[g]
        return gq * (sum(r * P + r * r / 2 for r in s.branch_lens[g]) + 300 * P)
    g = min(range(s.num_groups), key=cost)
    if cost(g) <= PROMPT_KEY_BUDGET:
        p0, p1 = int(s.cu_prompt[g]), int(s.cu_prompt[g + 1])
        rows = sorted({p1 - 1, max(p0, p1 - 50), max(p0, p1 - 299)})
        ref = S.key_rows(t, "prompt", rows, 0)
        idx = torch.tensor(rows, device="cuda")
        gk = _host(out["dk_p"].index_select(0, idx)[:, 0])
        gv = _host(out["dv_p"].index_select(0, idx)[:, 0])
        ek, ev = rel(gk, ref["dk"]), rel(gv, ref["dv"])
        log(f"[fullsize] {name} group {g} prompt keys: dK {ek:.2e} dV {ev:.2e}")
        assert ek <= TOL_GRAD and ev <= TOL_GRAD
    else:
        log(f"[fullsize] {name}: prompt-key reference over budget ({cost(g):.2e}); identity check only")

    # ---- identity: sum of dV over a group's keys == sum of dO over its query rows and heads
    dvp = out["dv_p"].double()
    dvr = out["dv_r"].double()
    dop = x["do_p"].double()
    dor = x["do_r"].double()
    for g in range(s.num_groups):
        p0, p1 = int(s.cu_prompt[g]), int(s.cu_prompt[g + 1])
        r0, r1 = int(s.cu_resp[s.cu_branch[g]]), int(s.cu_resp[s.cu_branch[g + 1]])
        lhs = dvp[p0:p1].sum(0) + dvr[r0:r1].sum(0)                                   # [Hkv, d]
        rhs = (dop[p0:p1].sum(0) + dor[r0:r1].sum(0)).view(s.num_kv_heads, gq, s.head_dim).sum(1)
        e = rel(lhs.cpu().numpy(), rhs.cpu().numpy())
        assert e <= TOL_GRAD, (g, e)
    log(f"[fullsize] {name}: dV-total identity holds for {s.num_groups} groups")
    del step, x, out
    torch.cuda.empty_cache()
