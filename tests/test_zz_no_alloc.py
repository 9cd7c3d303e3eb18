"""The allocation-free backward entry point (augtree_tree_bwd_noalloc,
through the C ABI): bitwise the outputs of augtree_tree_bwd on two calls in a
row, the second on a smaller batch (the device array keeps the first call's
contents); a batch beyond its fixed size rejected on the host; the unchunked
schedule when the chunks' partials do not fit; and a call captured in a graph
and replayed."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2609_33133_amd import _lib, api
from paper_2609_33133_amd import inputs as I
from paper_2609_33133_amd.api import GroupBatch
from paper_2609_33133_amd.group_attention import upload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _both(shape, seed, f32):
    gi = I.make_inputs(shape, seed=seed, qk_mult=1.0)
    b = GroupBatch.from_shape(shape)
    x = upload(gi)
    o_p, lse_p, o_r, lse_r, _, _ = api.tree_fwd(b, x["q_p"], x["k_p"], x["v_p"], x["q_r"], x["k_r"], x["v_r"])
    args = (x["q_p"], x["k_p"], x["v_p"], o_p, lse_p, x["do_p"], x["q_r"], x["k_r"], x["v_r"], o_r, lse_r, x["do_r"])
    ref = api.tree_bwd(b, *args, want_f32=f32)
    outs = [torch.full_like(t, 7) for t in ref[:6]]
    f32_out = torch.full((2, b.tp, b.hkv, b.d), 7.0, device="cuda") if f32 else None
    lib = _lib.load()
    P = api._ptr
    st = lib.augtree_tree_bwd_noalloc(b.ref, *(P(t) for t in args), P(outs[0]), P(outs[1]), P(outs[2]), P(f32_out),
                                      P(outs[3]), P(outs[4]), P(outs[5]), api._stream(None))
    _lib.check(st, "tree_bwd_noalloc")
    torch.cuda.synchronize()
    names = ("dq_p", "dk_p", "dv_p", "dq_r", "dk_r", "dv_r")
    for n, a, r in zip(names, outs, ref[:6]):
        assert torch.equal(a.view(torch.int16), r.view(torch.int16)), n
    if f32:
        assert torch.equal(f32_out, ref[6])


def test_noalloc_matches_tree_bwd_on_two_calls():
    big = I.custom_shape([700, 130, 256], [[5] * 12, [200, 129], [17] * 4], 8, 2, 128)   # > 32 tiles: schedule in the array
    small = I.custom_shape([90], [[65, 40]], 8, 2, 128)
    _both(big, 71, f32=True)
    _both(small, 72, f32=False)


def test_noalloc_rejects_batches_beyond_its_array():
    lib = _lib.load()
    cap = lib.augtree_noalloc_scratch_bytes()
    assert cap == 64 << 20
    # D alone needs (T_P + T_R) * Hq * 4 bytes: 2^20 rows x 32 heads = 128 MiB
    shape = I.custom_shape([1 << 19], [[1 << 19]], 32, 8, 128)
    b = GroupBatch.from_shape(shape)
    assert b.workspace_size(api.OP_TREE_BWD) > cap
    p = ctypes.c_void_p(1 << 20)
    st = lib.augtree_tree_bwd_noalloc(b.ref, *([p] * 15), None, p, p, p, None)
    assert st == _lib.AUGTREE_ERR_WORKSPACE
    assert "allocation-free" in lib.augtree_last_error().decode()


def _run_noalloc(b, args, outs, f32_out=None):
    lib = _lib.load()
    P = api._ptr
    return lib.augtree_tree_bwd_noalloc(b.ref, *(P(t) for t in args), P(outs[0]), P(outs[1]), P(outs[2]),
                                        P(f32_out), P(outs[3]), P(outs[4]), P(outs[5]), api._stream(None))


NAMES = ("dq_p", "dk_p", "dv_p", "dq_r", "dk_r", "dv_r")


def test_noalloc_runs_unchunked_when_the_chunks_do_not_fit():
    """Chunks of 3 query blocks make the tree backward's fp32 partials of this
    batch (P = 8192) exceed the 64 MiB array; the allocation-free call then
    runs one sweep per prompt-key tile: dQ and the branch-key gradients are
    bitwise those of augtree_tree_bwd, the prompt-key gradient the same sum in
    another fp32 order."""
    shape = I.custom_shape([8192], [[600, 350]], 8, 2, 128)
    gi = I.make_inputs(shape, seed=73, qk_mult=1.0)
    b = GroupBatch.from_shape(shape)
    x = upload(gi)
    o_p, lse_p, o_r, lse_r, _, _ = api.tree_fwd(b, x["q_p"], x["k_p"], x["v_p"], x["q_r"], x["k_r"], x["v_r"])
    args = (x["q_p"], x["k_p"], x["v_p"], o_p, lse_p, x["do_p"], x["q_r"], x["k_r"], x["v_r"], o_r, lse_r, x["do_r"])
    api.set_tree_chunk_blocks(3)
    try:
        assert b.workspace_size(api.OP_TREE_BWD) > _lib.load().augtree_noalloc_scratch_bytes()
        ref = api.tree_bwd(b, *args, want_f32=True)
        outs = [torch.full_like(t, 7) for t in ref[:6]]
        f32_out = torch.full((2, b.tp, b.hkv, b.d), 7.0, device="cuda")
        _lib.check(_run_noalloc(b, args, outs, f32_out), "tree_bwd_noalloc")
    finally:
        api.set_tree_chunk_blocks(0)
    torch.cuda.synchronize()
    for n, a, r in zip(NAMES, outs, ref[:6]):
        if n in ("dk_p", "dv_p"):
            continue
        assert torch.equal(a.view(torch.int16), r.view(torch.int16)), n
    e = (f32_out.double() - ref[6].double()).norm() / ref[6].double().norm()
    assert float(e) < 1e-5, float(e)
    assert torch.equal(f32_out[0].to(torch.bfloat16), outs[1]) and torch.equal(f32_out[1].to(torch.bfloat16), outs[2])


def test_noalloc_in_a_captured_graph():
    """A batch whose every launch carries its schedule in the kernel arguments
    enqueues kernels only: the allocation-free call captured once in a graph
    and replayed three times, with eager work between the replays, gives the
    eager outputs every time."""
    shape = I.custom_shape([256], [[128, 128]], 4, 4, 64)
    gi = I.make_inputs(shape, seed=74, qk_mult=1.0)
    b = GroupBatch.from_shape(shape)
    x = upload(gi)
    o_p, lse_p, o_r, lse_r, _, _ = api.tree_fwd(b, x["q_p"], x["k_p"], x["v_p"], x["q_r"], x["k_r"], x["v_r"])
    args = (x["q_p"], x["k_p"], x["v_p"], o_p, lse_p, x["do_p"], x["q_r"], x["k_r"], x["v_r"], o_r, lse_r, x["do_r"])
    ref = api.tree_bwd(b, *args)
    outs = [torch.full_like(t, 7) for t in ref[:6]]
    _lib.check(_run_noalloc(b, args, outs), "tree_bwd_noalloc")   # first call on the device: outside the capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        st = _run_noalloc(b, args, outs)
    _lib.check(st, "tree_bwd_noalloc (captured)")
    for _ in range(3):
        for t in outs:
            t.fill_(7)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for n, a, r in zip(NAMES, outs, ref[:6]):
            assert torch.equal(a.view(torch.int16), r.view(torch.int16)), n
