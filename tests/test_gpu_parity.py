"""GPU parity: every entry point of the C ABI against the fp64 oracle on the
same seeded bf16 inputs (small shapes that span several tiles and a ragged
tail; edge cases; closed-form mask probe; determinism; fused vs split)."""
import numpy as np
import pytest
import torch

from oracle import attention as A
from paper_2609_33133_amd import api
from paper_2609_33133_amd import inputs as I
from paper_2609_33133_amd.api import REPLAY_FUSED, REPLAY_SPLIT, GroupBatch
from paper_2609_33133_amd.group_attention import SharedStep, upload

from gpu_helpers import assert_close, log, oracle, rel, run_flattened, run_shared, to_np

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_33133_amd import _lib
    lib = _lib.load()
    assert lib.augtree_check_device() == 0, lib.augtree_last_error()


@pytest.mark.parametrize("path", ["tree", "calls"])
@pytest.mark.parametrize("mode", [REPLAY_FUSED, REPLAY_SPLIT])
def test_tiny_workload_full_parity(mode, path):
    gi = I.make_config("tiny")
    ref = oracle(gi)
    got, _ = run_shared(gi, mode=mode, path=path)
    assert_close(got, ref, f"tiny mode={mode} path={path}")


SHAPES = [
    # (prompt lens, branch lens, hq, hkv, d, qk_mult)
    ([300], [[200, 77, 129]], 8, 2, 128, None),
    ([130, 64], [[1, 65], [128, 3, 200]], 4, 4, 64, None),
    ([257], [[31, 256]], 8, 2, 128, 1.0),            # sharp logits
    ([1, 2], [[1, 300], [5]], 4, 1, 128, 1.0),        # P = 1, R = 1, MQA
    ([64, 128, 192], [[64], [128], [192, 1]], 8, 2, 64, 1.0),
    ([500], [[40, 41, 42, 43]], 4, 2, 128, 4.0),      # very sharp
    ([200, 33], [[100, 37, 64], [5]], 28, 4, 128, None),   # 28 / 4 heads: g = 7
    ([130], [[70, 1, 129]], 28, 4, 128, 1.0),              # g = 7, sharp
    ([96], [[3 + (7 * i) % 20 for i in range(64)]], 8, 2, 64, None),  # G = 64 short branches
    ([200], [[100, 50]], 16, 2, 128, None),                # g = 8
    ([150, 70], [[64, 129], [200]], 8, 8, 128, 1.0),       # g = 1 at d = 128, sharp
    ([1], [[1000]], 4, 1, 64, 1.0),                        # one-token prompt, long branch, d = 64
]


@pytest.mark.parametrize("case", range(len(SHAPES)))
def test_small_shapes(case):
    ps, rs, hq, hkv, d, mult = SHAPES[case]
    shape = I.custom_shape(ps, rs, hq, hkv, d)
    gi = I.make_inputs(shape, seed=100 + case, qk_mult=mult)
    log(f"case {case}: P={ps} R={rs} hq={hq} hkv={hkv} d={d} mult={mult}")
    ref = oracle(gi)
    for path in ("tree", "calls"):
        for mode in (REPLAY_FUSED, REPLAY_SPLIT):
            got, _ = run_shared(gi, mode=mode, path=path)
            assert_close(got, ref, f"case {case} mode {mode} path {path}")


@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_random_ragged_shapes(seed):
    rng = np.random.default_rng(1000 + seed)
    shape = I.random_shape(rng, max_groups=3, max_p=400, max_g=4, max_r=300,
                           heads=((4, 4, 64), (8, 2, 128), (4, 1, 128)))
    gi = I.make_inputs(shape, seed=2000 + seed, qk_mult=1.0 if seed % 2 else None)
    log(f"seed {seed}: P={shape.prompt_lens} R={shape.branch_lens} h={shape.num_q_heads}/{shape.num_kv_heads} "
        f"d={shape.head_dim}")
    ref = oracle(gi)
    got, _ = run_shared(gi, n_seed=1 + seed, path="calls")
    assert_close(got, ref, f"random {seed} calls n_seed={1 + seed}")
    got, _ = run_shared(gi, mode=api.REPLAY_AUTO)
    assert_close(got, ref, f"random {seed} tree auto")


def test_q_zero_probe_closed_form():
    """Q = 0: LSE = ln(#visible keys), O[..., 0] = mean of visible position labels."""
    shape = I.custom_shape([100, 37], [[64, 1, 100], [20, 90]], 8, 2, 128)
    gi = I.make_inputs(shape, seed=7)
    gi.q_p[:] = 0
    gi.q_r[:] = 0
    for g in range(shape.num_groups):
        p0, p1 = shape.cu_prompt[g], shape.cu_prompt[g + 1]
        gi.v_p[p0:p1, :, 0] = I.f32_to_bf16_bits(np.arange(p1 - p0, dtype=np.float32))[:, None]
        for b in range(shape.cu_branch[g], shape.cu_branch[g + 1]):
            r0, r1 = shape.cu_resp[b], shape.cu_resp[b + 1]
            gi.v_r[r0:r1, :, 0] = I.f32_to_bf16_bits((p1 - p0 + np.arange(r1 - r0)).astype(np.float32))[:, None]
    for mode, path in ((REPLAY_FUSED, "tree"), (REPLAY_SPLIT, "tree"), (REPLAY_FUSED, "calls")):
        got, _ = run_shared(gi, mode=mode, path=path)
        for g in range(shape.num_groups):
            p0, p1 = shape.cu_prompt[g], shape.cu_prompt[g + 1]
            P = p1 - p0
            pos = np.arange(P)
            assert np.max(np.abs(got["lse_p"][:, p0:p1] - np.log(pos + 1))) < 1e-5
            assert rel(got["o_p"][p0:p1, :, 0], np.broadcast_to((pos / 2)[:, None], (P, 8))) < 1e-2
            for b in range(shape.cu_branch[g], shape.cu_branch[g + 1]):
                r0, r1 = shape.cu_resp[b], shape.cu_resp[b + 1]
                t = np.arange(r1 - r0)
                assert np.max(np.abs(got["lse_r"][:, r0:r1] - np.log(P + t + 1))) < 1e-5
                want = np.broadcast_to(((P + t) / 2)[:, None], (r1 - r0, 8))
                assert rel(got["o_r"][r0:r1, :, 0], want) < 1e-2


def test_rising_logits_move_the_softmax_reference():
    """Logits that rise along the key positions, at a different slope per
    query head: the running row maximum of the online softmax grows on every
    64-key block, by steps below and above the forward kernel's rescale
    margin (2^8), and never (negative slope). The ramp sits in component 0:
    key j has k[0] = j / 640 and query head h has q[0] = slope_h. (A steeper
    key ramp with flatter slopes gives the same logits but a large common
    k[0] over the keys that carry the softmax mass, whose cancellation in
    dQ = s dS K amplifies the bf16 rounding of dS beyond the tolerance.)"""
    shape = I.custom_shape([700], [[150, 90]], 8, 2, 128)
    gi = I.make_inputs(shape, seed=11)
    P = shape.prompt_lens[0]
    # log2-unit rise per 64 keys = slope * 64 / 640 * scale * log2(e) ~ 0.01275 * slope
    slopes = np.array([0.0, 40.0, 160.0, 400.0, 640.0, 1000.0, 1570.0, -300.0], np.float32)
    gi.q_p[:, :, 0] = I.f32_to_bf16_bits(np.broadcast_to(slopes, (P, 8)).copy())
    gi.q_r[:, :, 0] = I.f32_to_bf16_bits(np.broadcast_to(slopes, (gi.q_r.shape[0], 8)).copy())
    gi.k_p[:, :, 0] = I.f32_to_bf16_bits((np.arange(P, dtype=np.float32) / 640)[:, None].repeat(2, 1))
    for b in range(2):
        r0, r1 = shape.cu_resp[b], shape.cu_resp[b + 1]
        pos = (P + np.arange(r1 - r0, dtype=np.float32)) / 640
        gi.k_r[r0:r1, :, 0] = I.f32_to_bf16_bits(pos[:, None].repeat(2, 1))
    ref = oracle(gi)
    for mode, path in ((REPLAY_FUSED, "tree"), (REPLAY_SPLIT, "tree"), (REPLAY_FUSED, "calls")):
        got, _ = run_shared(gi, mode=mode, path=path)
        assert_close(got, ref, f"rising logits mode {mode} path {path}")


def test_fused_equals_split():
    shape = I.custom_shape([333, 70], [[100, 200], [65, 1, 129]], 8, 2, 128)
    gi = I.make_inputs(shape, seed=8, qk_mult=1.0)
    a, _ = run_shared(gi, mode=REPLAY_FUSED)
    b, _ = run_shared(gi, mode=REPLAY_SPLIT)
    assert rel(a["o_r"], b["o_r"]) < 2e-3
    assert np.max(np.abs(a["lse_r"] - b["lse_r"])) < 1e-4
    for k in ("dq_r", "dk_r", "dv_r", "dk_p", "dv_p"):
        assert rel(a[k], b[k]) < 5e-3, k


@pytest.mark.parametrize("path", ["tree", "calls"])
def test_determinism_bitwise(path):
    shape = I.custom_shape([300, 90], [[100, 200, 5], [65, 129]], 8, 2, 128)
    gi = I.make_inputs(shape, seed=9)
    b = GroupBatch.from_shape(shape)
    x = upload(gi)
    outs = []
    for _ in range(3):
        step = SharedStep(b, "cuda", n_seed=3, path=path)
        step.run(x)
        torch.cuda.synchronize()
        outs.append({k: v.clone() for k, v in step.outputs().items()})
    for o in outs[1:]:
        for k in o:
            assert torch.equal(o[k].view(torch.uint8) if o[k].dtype != torch.float32 else o[k],
                               outs[0][k].view(torch.uint8) if o[k].dtype != torch.float32 else outs[0][k]), k


def _bits(t: torch.Tensor) -> torch.Tensor:
    return t.contiguous().view(torch.uint8)


def _batch_of(parts):
    """Inputs of a batch made of single-tree inputs, in the given order."""
    s0 = parts[0].shape
    shape = I.custom_shape([p.shape.prompt_lens[0] for p in parts], [list(p.shape.branch_lens[0]) for p in parts],
                           s0.num_q_heads, s0.num_kv_heads, s0.head_dim)
    fields = {n: np.concatenate([getattr(p, n) for p in parts]) for n in
              ("q_p", "k_p", "v_p", "q_r", "k_r", "v_r", "do_p", "do_r")}
    return I.GroupInputs(shape=shape, **fields)


def _run_step(gi, prefill_bwd_first=False, path="calls"):
    b = GroupBatch.from_shape(gi.shape)
    step = SharedStep(b, "cuda", mode=REPLAY_FUSED, n_seed=2, path=path)
    x = upload(gi)
    step.forward(x)
    if prefill_bwd_first:
        api.prefill_bwd(b, x["q_p"], x["k_p"], x["v_p"], step.o_p, step.lse_p, x["do_p"], step.dq_p, None,
                        step.dkv_self, ws=step.ws["pb"])
        api.replay_bwd(b, x["q_r"], x["k_r"], x["v_r"], x["k_p"], x["v_p"], step.o_r, step.lse_r, x["do_r"],
                       step.n_seed, step.dq_r, step.dk_r, step.dv_r, step.seed, ws=step.ws["rb"])
        api.prompt_grad_reduce(step.seed, self_part=step.dkv_self, out=step.dkv_p)
    else:
        step.backward(x)
    torch.cuda.synchronize()
    return {k: v.clone() for k, v in step.outputs().items()}


def test_outputs_independent_of_batch_and_call_order():
    """A tree's outputs are bitwise the same alone, first or second in a batch
    (different tile schedules: the tiles of the other tree are interleaved or
    ordered around them) and with the two backward calls in either order: every
    output element is computed by one workgroup in a fixed order, and the
    Eq. 2 sum runs in a fixed order (no atomics)."""
    a = I.make_inputs(I.custom_shape([300], [[100, 200, 5]], 8, 2, 128), seed=21, qk_mult=1.0)
    b = I.make_inputs(I.custom_shape([90], [[65, 129]], 8, 2, 128), seed=22)
    alone = _run_step(a)
    swapped = _run_step(a, prefill_bwd_first=True)
    for k in alone:
        assert torch.equal(_bits(swapped[k]), _bits(alone[k])), f"call order: {k}"
    tp_a, tr_a, tp_b, tr_b = 300, 305, 90, 194
    for parts, p0, r0 in (([a, b], 0, 0), ([b, a], tp_b, tr_b)):
        got = _run_step(_batch_of(parts))
        _same_rows(got, alone, p0, r0, tp_a, tr_a)
    alone = _run_step(a, path="tree")
    for parts, p0, r0 in (([a, b], 0, 0), ([b, a], tp_b, tr_b)):
        _same_rows(_run_step(_batch_of(parts), path="tree"), alone, p0, r0, tp_a, tr_a)


def _same_rows(got, alone, p0, r0, tp_a, tr_a):
    """The rows of tree `a` inside a batch output are bitwise its outputs alone."""
    rows = {"o_p": (p0, tp_a), "dq_p": (p0, tp_a), "dk_p": (p0, tp_a), "dv_p": (p0, tp_a),
            "o_r": (r0, tr_a), "dq_r": (r0, tr_a), "dk_r": (r0, tr_a), "dv_r": (r0, tr_a)}
    for k, (o, n) in rows.items():
        assert torch.equal(_bits(got[k][o:o + n]), _bits(alone[k])), f"batch position {p0}: {k}"
    assert torch.equal(_bits(got["lse_p"][:, p0:p0 + tp_a]), _bits(alone["lse_p"])), "lse_p"
    assert torch.equal(_bits(got["lse_r"][:, r0:r0 + tr_a]), _bits(alone["lse_r"])), "lse_r"


@pytest.mark.parametrize("n_seed", [1, 2, 5])
def test_seed_chunks_give_same_prompt_gradient(n_seed):
    shape = I.custom_shape([200], [[150, 150, 40, 300]], 8, 2, 128)
    gi = I.make_inputs(shape, seed=10)
    ref = oracle(gi)
    got, step = run_shared(gi, n_seed=n_seed, path="calls")
    assert_close(got, ref, f"n_seed={n_seed}")
    # every slab holds its chunk's contribution; their sum is the branch total
    sh = A.shared_fwd_bwd(shape.cu_prompt, shape.cu_branch, shape.cu_resp, 8, 2, shape.scale,
                          *(I.bf16_bits_to_f64(getattr(gi, n)) for n in ("q_p", "k_p", "v_p", "q_r", "k_r", "v_r",
                                                                          "do_p", "do_r")))
    seeds = to_np(step.seed).sum(0)
    assert rel(seeds[0], sh["seed_k"].sum(0)) < 2e-2
    assert rel(seeds[1], sh["seed_v"].sum(0)) < 2e-2
    assert rel(to_np(step.dkv_self[0]), sh["dk_p_self"]) < 2e-2


def test_lse_merge_entry_point():
    rng = np.random.default_rng(11)
    n, rows, heads, d = 3, 257, 4, 64
    o = rng.standard_normal((n, rows, heads, d)).astype(np.float32)
    l = (rng.standard_normal((n, heads, rows)) * 3).astype(np.float32)
    l[1, 0, :50] = -np.inf                  # an empty part
    l[:, 1, 7] = -np.inf                    # a row with every part empty
    to = torch.from_numpy(o).cuda()
    tl = torch.from_numpy(l).cuda()
    ob, of, lse = api.lse_merge(to, tl)
    ob2, of2, lse2 = api.lse_merge(to, tl, want_bf16=False)
    torch.cuda.synchronize()
    ro, rl = A.lse_merge(o.astype(np.float64).transpose(0, 2, 1, 3), l.astype(np.float64))
    ro = ro.transpose(1, 0, 2)
    got_f = to_np(of2)
    got_l = to_np(lse2)
    fin = np.isfinite(rl)
    assert np.array_equal(np.isfinite(got_l), fin)
    assert np.max(np.abs(got_l[fin] - rl[fin])) < 1e-5
    assert np.all(got_f[7, 1] == 0)
    assert rel(got_f, ro) < 1e-5
    assert rel(to_np(ob), ro) < 1e-2


def test_prompt_grad_reduce_bitexact_fp32():
    """fp32 sum in index order (self first): equal bit for bit to the same
    sequence of float32 additions on the host."""
    rng = np.random.default_rng(12)
    n, rows, heads, d = 5, 300, 2, 64
    parts = rng.standard_normal((n, 2, rows, heads, d)).astype(np.float32)
    selfp = rng.standard_normal((2, rows, heads, d)).astype(np.float32)
    out_b, out_f = api.prompt_grad_reduce(torch.from_numpy(parts).cuda(), self_part=torch.from_numpy(selfp).cuda(),
                                          want_bf16=False)
    torch.cuda.synchronize()
    exp = selfp.copy()
    for k in range(n):
        exp = (exp + parts[k]).astype(np.float32)
    assert np.array_equal(out_f.cpu().numpy(), exp)
    # row map over one shared slab, with absent rows
    slab = rng.standard_normal((2, 50, heads, d)).astype(np.float32)
    rm = np.full((3, 20), -1, np.int32)
    rm[0] = np.arange(20)
    rm[1, :10] = np.arange(30, 40)
    rm[2, 5:] = np.arange(35, 50)
    _, got = api.prompt_grad_reduce(torch.from_numpy(slab).cuda(), row_map=torch.from_numpy(rm).cuda(), rows=20,
                                    shared_slab=True, n_parts=3, want_bf16=False)
    torch.cuda.synchronize()
    exp = np.zeros((2, 20, heads, d), np.float32)
    for k in range(3):
        for r in range(20):
            if rm[k, r] >= 0:
                exp[:, r] = (exp[:, r] + slab[:, rm[k, r]]).astype(np.float32)
    assert np.array_equal(got.cpu().numpy(), exp)


def test_prefill_bwd_fp32_dq_matches_bf16():
    shape = I.custom_shape([190, 64], [[1], [1]], 8, 2, 128)
    gi = I.make_inputs(shape, seed=13)
    b = GroupBatch.from_shape(shape)
    x = upload(gi)
    o, lse = api.prefill_fwd(b, x["q_p"], x["k_p"], x["v_p"])
    dqb, _, s1 = api.prefill_bwd(b, x["q_p"], x["k_p"], x["v_p"], o, lse, x["do_p"])
    _, dqf, s2 = api.prefill_bwd(b, x["q_p"], x["k_p"], x["v_p"], o, lse, x["do_p"], want_bf16=False)
    torch.cuda.synchronize()
    assert torch.equal(dqf.to(torch.bfloat16), dqb)
    assert torch.equal(s1, s2)


def test_flattened_baseline_matches_oracle():
    shape = I.custom_shape([150, 60], [[100, 33], [20, 64, 7, 129]], 8, 2, 128)
    gi = I.make_inputs(shape, seed=14, qk_mult=1.0)
    ref = oracle(gi)
    got = run_flattened(gi)
    assert_close(got, ref, "flattened")


def test_auto_mode_mixed_groups():
    """AUGTREE_REPLAY_AUTO runs short-branch groups SPLIT and long-branch
    groups FUSED in one call; every output against the oracle."""
    shape = I.custom_shape([700, 130, 256], [[5] * 12, [200, 129], [17] * 4], 8, 2, 128)
    b = GroupBatch.from_shape(shape)
    assert api.replay_split_groups(b).tolist() == [1, 0, 1]
    gi = I.make_inputs(shape, seed=41, qk_mult=1.0)
    ref = oracle(gi)
    for path in ("tree", "calls"):
        got, _ = run_shared(gi, mode=api.REPLAY_AUTO, path=path)
        assert_close(got, ref, f"auto mixed {path}")


@pytest.mark.parametrize("ps,rs,same_as", [([300], [[250, 260]], REPLAY_FUSED), ([1000], [[3] * 20], REPLAY_SPLIT)])
def test_auto_mode_equals_chosen_mode_bitwise(ps, rs, same_as):
    shape = I.custom_shape(ps, rs, 8, 2, 128)
    gi = I.make_inputs(shape, seed=42)
    a, _ = run_shared(gi, mode=api.REPLAY_AUTO)
    m, _ = run_shared(gi, mode=same_as)
    for k in ("o_r", "lse_r"):
        assert np.array_equal(a[k], m[k]), k
