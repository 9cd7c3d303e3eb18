"""The two-call form of a step (augtree_tree_fwd + augtree_tree_bwd) against
the six separate entry points on the same inputs: the forward outputs, dQ and
the branch-key gradients come from the same per-tile arithmetic and must be
bitwise equal; the prompt-key gradient (Eq. 2) is the same sum in another
fp32 order (registers in one sweep vs two fp32 partial sums added by
prompt_grad_reduce), so its fp32 values agree to fp32 rounding."""
import numpy as np
import pytest
import torch

from paper_2609_33133_amd import api
from paper_2609_33133_amd import inputs as I
from paper_2609_33133_amd.api import REPLAY_AUTO, REPLAY_FUSED, REPLAY_SPLIT, GroupBatch
from paper_2609_33133_amd.group_attention import SharedStep, upload

from gpu_helpers import assert_close, log, oracle, rel, run_shared

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


CASES = [
    # prompt lens, branch lens, hq, hkv, d, mode
    ([300, 70], [[200, 77, 129], [1, 64]], 8, 2, 128, REPLAY_FUSED),
    ([130, 64], [[1, 65], [128, 3, 200]], 4, 4, 64, REPLAY_SPLIT),
    ([700, 130, 256], [[5] * 12, [200, 129], [17] * 4], 8, 2, 128, REPLAY_AUTO),
    ([1000], [[40] * 24], 28, 4, 128, REPLAY_FUSED),   # > 32 tiles per launch: schedules in the workspace
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_tree_calls_match_separate_calls(case):
    ps, rs, hq, hkv, d, mode = CASES[case]
    shape = I.custom_shape(ps, rs, hq, hkv, d)
    gi = I.make_inputs(shape, seed=500 + case, qk_mult=1.0)
    b = GroupBatch.from_shape(shape)
    x = upload(gi)
    tree = SharedStep(b, "cuda", mode=mode, path="tree")
    calls = SharedStep(b, "cuda", mode=mode, n_seed=1, path="calls")
    tree.run(x)
    calls.run(x)
    # fp32 prompt-key gradient of the tree call
    f32 = api.tree_bwd(b, x["q_p"], x["k_p"], x["v_p"], tree.o_p, tree.lse_p, x["do_p"], x["q_r"], x["k_r"],
                       x["v_r"], tree.o_r, tree.lse_r, x["do_r"], want_f32=True)[6]
    _, calls_f32 = api.prompt_grad_reduce(calls.seed, self_part=calls.dkv_self, want_bf16=False)
    torch.cuda.synchronize()
    a, c = tree.outputs(), calls.outputs()
    for k in ("o_p", "lse_p", "o_r", "lse_r", "dq_p", "dq_r", "dk_r", "dv_r"):
        assert torch.equal(a[k].contiguous().view(torch.uint8), c[k].contiguous().view(torch.uint8)), k
    e = rel(f32.double().cpu().numpy(), calls_f32.double().cpu().numpy())
    log(f"[tree vs calls] case {case}: prompt dK/dV fp32 rel diff {e:.2e}")
    assert e < 1e-5
    # the bf16 outputs are the fp32 values rounded once
    assert torch.equal(f32[0].to(torch.bfloat16), a["dk_p"]) and torch.equal(f32[1].to(torch.bfloat16), a["dv_p"])
    for k in ("dk_p", "dv_p"):
        assert rel(a[k].double().cpu().numpy(), c[k].double().cpu().numpy()) < 5e-3, k


def test_tree_bwd_rejects_bad_arguments():
    shape = I.custom_shape([10], [[4, 5]], 4, 2, 64)
    gi = I.make_inputs(shape, seed=1)
    b = GroupBatch.from_shape(shape)
    x = upload(gi)
    o_p, lse_p, o_r, lse_r, _, _ = api.tree_fwd(b, x["q_p"], x["k_p"], x["v_p"], x["q_r"], x["k_r"], x["v_r"])
    with pytest.raises(ValueError):
        api.tree_bwd(b, x["q_p"], x["k_p"], x["v_p"], o_p, lse_p, x["do_p"], x["q_r"], x["k_r"], x["v_r"], o_r,
                     lse_r, x["do_r"], dq_p=torch.empty((9, 4, 64), dtype=torch.bfloat16, device="cuda"))
    lib = api._lib.load()
    st = lib.augtree_tree_bwd(b.ref, *([None] * 19), None, 0, None)
    assert st == 1 and "null pointer" in lib.augtree_last_error().decode()


@pytest.mark.parametrize("case,chunk", [(0, 3), (1, 3), (2, 3), (3, 3), (0, 1)])
def test_tree_chunked_prompt_sweeps(case, chunk):
    """Prompt-key sweeps cut into chunks (3 query blocks each, so every group
    with more than 3 x 64 / g branch rows is chunked; with 1 block the chunk
    edges round to 64-row multiples and many chunks are empty, their partials
    zero): dQ and the branch-key gradients are bitwise those of the six
    separate calls, the prompt-key gradient agrees with the six-call and the
    unchunked sums to fp32 rounding, and its bf16 output is its fp32 value
    rounded once."""
    ps, rs, hq, hkv, d, mode = CASES[case]
    shape = I.custom_shape(ps, rs, hq, hkv, d)
    gi = I.make_inputs(shape, seed=700 + case, qk_mult=1.0)
    b = GroupBatch.from_shape(shape)
    x = upload(gi)
    plain = SharedStep(b, "cuda", mode=mode, path="tree")
    plain.run(x)
    f32_plain = api.tree_bwd(b, x["q_p"], x["k_p"], x["v_p"], plain.o_p, plain.lse_p, x["do_p"], x["q_r"],
                             x["k_r"], x["v_r"], plain.o_r, plain.lse_r, x["do_r"], want_f32=True)[6]
    api.set_tree_chunk_blocks(chunk)
    try:
        tree = SharedStep(b, "cuda", mode=mode, path="tree")
        tree.run(x)
        f32 = api.tree_bwd(b, x["q_p"], x["k_p"], x["v_p"], tree.o_p, tree.lse_p, x["do_p"], x["q_r"], x["k_r"],
                           x["v_r"], tree.o_r, tree.lse_r, x["do_r"], want_f32=True)[6]
    finally:
        api.set_tree_chunk_blocks(0)
    calls = SharedStep(b, "cuda", mode=mode, n_seed=1, path="calls")
    calls.run(x)
    _, calls_f32 = api.prompt_grad_reduce(calls.seed, self_part=calls.dkv_self, want_bf16=False)
    torch.cuda.synchronize()
    a = {k: v.clone() for k, v in tree.outputs().items()}
    c = calls.outputs()
    for k in ("o_p", "lse_p", "o_r", "lse_r", "dq_p", "dq_r", "dk_r", "dv_r"):
        assert torch.equal(a[k].contiguous().view(torch.uint8), c[k].contiguous().view(torch.uint8)), k
    e_calls = rel(f32.double().cpu().numpy(), calls_f32.double().cpu().numpy())
    e_plain = rel(f32.double().cpu().numpy(), f32_plain.double().cpu().numpy())
    log(f"[tree chunks] case {case} chunk {chunk}: prompt dK/dV fp32 rel diff vs calls {e_calls:.2e}, "
        f"vs unchunked {e_plain:.2e}")
    assert e_calls < 1e-5 and e_plain < 1e-5
    assert torch.equal(f32[0].to(torch.bfloat16), a["dk_p"]) and torch.equal(f32[1].to(torch.bfloat16), a["dv_p"])
    # a second run gives the same bits
    api.set_tree_chunk_blocks(chunk)
    try:
        tree.run(x)
    finally:
        api.set_tree_chunk_blocks(0)
    torch.cuda.synchronize()
    a2 = tree.outputs()
    for k in ("dk_p", "dv_p", "dq_p", "dq_r"):
        assert torch.equal(a[k].view(torch.uint8), a2[k].view(torch.uint8)), k


@pytest.mark.parametrize("seed", range(8))
def test_tree_random_shapes_against_oracle(seed):
    """Random ragged batches (up to 3 trees, 6 branches, GQA g = 1, 4, 7, 8,
    d = 64 and 128, normal and sharp logits) through the two-call step, with
    the default sweeps and with prompt-key sweeps cut into 3-block chunks,
    each against the fp64 oracle."""
    rng = np.random.default_rng(5000 + seed)
    shape = I.random_shape(rng, max_groups=3, max_p=700, max_g=6, max_r=500,
                           heads=((4, 4, 64), (8, 2, 128), (4, 1, 128), (28, 4, 128), (16, 2, 64), (8, 8, 128)))
    gi = I.make_inputs(shape, seed=6000 + seed, qk_mult=[None, 1.0, 2.0][seed % 3])
    log(f"[tree random] seed {seed}: P={shape.prompt_lens} R={shape.branch_lens} "
        f"h={shape.num_q_heads}/{shape.num_kv_heads} d={shape.head_dim}")
    ref = oracle(gi)
    for chunk in (0, 3):
        api.set_tree_chunk_blocks(chunk)
        try:
            got, _ = run_shared(gi, mode=REPLAY_AUTO)
        finally:
            api.set_tree_chunk_blocks(0)
        assert_close(got, ref, f"tree random {seed} chunk {chunk}")
