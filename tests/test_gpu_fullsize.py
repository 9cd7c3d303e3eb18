"""Full-size parity on the large workloads, in the launch configuration
bench.py times (the two-call tree step, fused replay), plus the six-call path
in split mode and with chunked prompt-key seeds.

The full fp64 oracle cannot run at these sizes, so the comparison uses
``oracle.sampled`` on chosen rows:
* query rows (first/last rows of groups and branches plus random rows) of
  three query heads (first, middle, last): O, LSE, dQ;
* key rows near the end of branches (dK_R, dV_R) of the first and last KV head;
* prompt key rows (dK_P, dV_P: the Eq. 2 total over the prompt queries and
  every branch) of the first and last KV head: early keys (positions 0, 127
  and 128: the longest causal sweeps and a key-tile edge) and late ones, on
  every workload (one or two groups of the ragged batch);
and an identity that holds at any size: for every group and KV head, the sum
of dV over all its keys (prompt and branches) equals the sum of dO over the
query rows and query heads that read them (each softmax row sums to one).
The prompt-key references run on a process pool (``oracle.sampled.key_rows``
with workers; the same bits as serial).
"""
import os
import time
import types

import numpy as np
import pytest
import torch

from oracle import sampled as S
from paper_2609_33133_amd import inputs as I
from paper_2609_33133_amd.api import REPLAY_FUSED, REPLAY_SPLIT, GroupBatch
from paper_2609_33133_amd.group_attention import SharedStep, upload

from gpu_helpers import TOL_GRAD, TOL_LSE, TOL_O, log, rel

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

# oracle worker processes: the CPU share of one GPU
WORKERS = max(1, min(16, len(os.sched_getaffinity(0))))


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


def _prompt_groups(s):
    """Groups whose prompt keys are compared: the only one, or (ragged) the
    cheapest group and the group with the most branches among the cheaper half."""
    gq = s.num_q_heads // s.num_kv_heads

    def cost(g):
        P = s.prompt_lens[g]
        return gq * (P * P / 2 + sum(r * (P + r) for r in s.branch_lens[g]))
    if s.num_groups == 1:
        return [0], cost
    order = sorted(range(s.num_groups), key=cost)
    cheap = order[: max(1, len(order) // 2)]
    many = max(cheap, key=lambda g: (len(s.branch_lens[g]), -cost(g)))
    return sorted({order[0], many}), cost


def _compare(name, gi, out, x, label):
    s = gi.shape
    t = types.SimpleNamespace(cu_prompt=s.cu_prompt, cu_branch=s.cu_branch, cu_resp=s.cu_resp,
                              num_q_heads=s.num_q_heads, num_kv_heads=s.num_kv_heads, head_dim=s.head_dim,
                              **{n: getattr(gi, n) for n in ("q_p", "k_p", "v_p", "q_r", "k_r", "v_r", "do_p",
                                                             "do_r")})
    rng = np.random.default_rng(123)
    groups = list(range(min(3, s.num_groups)))
    p_rows = _sample_rows(rng, [(int(s.cu_prompt[g]), int(s.cu_prompt[g + 1])) for g in groups], 6, s.total_prompt)
    br = [0, s.num_branches - 1, int(rng.integers(0, s.num_branches))]
    r_rows = _sample_rows(rng, [(int(s.cu_resp[i]), int(s.cu_resp[i + 1])) for i in br], 6, s.total_resp)
    kv_heads = sorted({0, s.num_kv_heads - 1})

    # ---- query rows
    for h in sorted({0, s.num_q_heads // 2, s.num_q_heads - 1}):
        for kind, rows, o, lse, dq in (("prompt", p_rows, "o_p", "lse_p", "dq_p"),
                                       ("resp", r_rows, "o_r", "lse_r", "dq_r")):
            ref = S.query_rows(t, kind, rows, h)
            idx = torch.tensor(rows, device="cuda")
            go = _host(out[o].index_select(0, idx)[:, h])
            gl = _host(out[lse][h].index_select(0, idx))
            gd = _host(out[dq].index_select(0, idx)[:, h])
            eo, el, ed = rel(go, ref["o"]), float(np.max(np.abs(gl - ref["lse"]))), rel(gd, ref["dq"])
            log(f"[fullsize] {label} {kind} rows head {h}: O {eo:.2e} LSE {el:.2e} dQ {ed:.2e}")
            assert eo <= TOL_O and el <= TOL_LSE and ed <= TOL_GRAD

    # ---- response keys near the end of branches
    for bi in br[:2]:
        r0, r1 = int(s.cu_resp[bi]), int(s.cu_resp[bi + 1])
        rows = sorted({max(r0, r1 - 1), max(r0, r1 - 37), max(r0, r1 - 200)})
        for kh in kv_heads:
            ref = S.key_rows(t, "resp", rows, kh, workers=WORKERS)
            idx = torch.tensor(rows, device="cuda")
            gk = _host(out["dk_r"].index_select(0, idx)[:, kh])
            gv = _host(out["dv_r"].index_select(0, idx)[:, kh])
            ek, ev = rel(gk, ref["dk"]), rel(gv, ref["dv"])
            log(f"[fullsize] {label} branch {bi} keys kv {kh}: dK {ek:.2e} dV {ev:.2e}")
            assert ek <= TOL_GRAD and ev <= TOL_GRAD

    # ---- prompt keys, early and late (Eq. 2 total: prompt queries + every branch)
    pgroups, cost = _prompt_groups(s)
    for g in pgroups:
        p0, p1 = int(s.cu_prompt[g]), int(s.cu_prompt[g + 1])
        rows = sorted({p0, min(p1 - 1, p0 + 127), min(p1 - 1, p0 + 128), max(p0, p1 - 50), p1 - 1})
        for kh in kv_heads:
            t0 = time.time()
            ref = S.key_rows(t, "prompt", rows, kh, workers=WORKERS)
            idx = torch.tensor(rows, device="cuda")
            gk = _host(out["dk_p"].index_select(0, idx)[:, kh])
            gv = _host(out["dv_p"].index_select(0, idx)[:, kh])
            ek, ev = rel(gk, ref["dk"]), rel(gv, ref["dv"])
            log(f"[fullsize] {label} group {g} prompt keys {[r - p0 for r in rows]} kv {kh}: dK {ek:.2e} dV {ev:.2e} "
                f"(reference {cost(g):.2e} row-key pairs, {time.time() - t0:.1f} s on {WORKERS} workers)")
            assert ek <= TOL_GRAD and ev <= TOL_GRAD

    # ---- identity: sum of dV over a group's keys == sum of dO over its query rows and heads
    gq = s.num_q_heads // s.num_kv_heads
    dvp, dvr = out["dv_p"].double(), out["dv_r"].double()
    dop, dor = x["do_p"].double(), x["do_r"].double()
    for g in range(s.num_groups):
        p0, p1 = int(s.cu_prompt[g]), int(s.cu_prompt[g + 1])
        r0, r1 = int(s.cu_resp[s.cu_branch[g]]), int(s.cu_resp[s.cu_branch[g + 1]])
        lhs = dvp[p0:p1].sum(0) + dvr[r0:r1].sum(0)                                   # [Hkv, d]
        rhs = (dop[p0:p1].sum(0) + dor[r0:r1].sum(0)).view(s.num_kv_heads, gq, s.head_dim).sum(1)
        e = rel(lhs.cpu().numpy(), rhs.cpu().numpy())
        assert e <= TOL_GRAD, (g, e)
    log(f"[fullsize] {label}: dV-total identity holds for {s.num_groups} groups")


def _run(name, mode=REPLAY_FUSED, path="tree", n_seed=None):
    log(f"[fullsize] {name} ({path}, mode {mode}): generating inputs")
    gi = I.make_config(name)
    b = GroupBatch.from_shape(gi.shape)
    x = upload(gi, "cuda")
    step = SharedStep(b, "cuda", mode=mode, n_seed=n_seed, path=path)
    log(f"[fullsize] {name}: running the hot path (n_seed={step.n_seed})")
    step.run(x)
    torch.cuda.synchronize()
    out = step.outputs()
    for k, v in out.items():
        assert torch.isfinite(v.float()).all(), k
    _compare(name, gi, out, x, f"{name}/{path}/mode{mode}")
    del step, x, out
    torch.cuda.empty_cache()


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["balanced", "prompt", "response", "ragged", "gsweep64", "prompt_gqa7"])
def test_fullsize_sampled(name):
    _run(name)


@pytest.mark.timeout(900)
def test_fullsize_six_calls_split():
    """The six separate entry points at full size, split replay (partials + merge)."""
    _run("balanced", mode=REPLAY_SPLIT, path="calls")


@pytest.mark.timeout(900)
def test_fullsize_six_calls_chunked_seeds():
    """The six separate entry points on the prompt-heavy tree with the branch
    rows' prompt-key gradient cut into 8 chunked seed slabs (chunk edges inside
    the branches) summed by prompt_grad_reduce."""
    _run("prompt", path="calls", n_seed=8)
