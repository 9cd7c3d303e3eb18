"""The C-ABI library loads, exports every symbol include/augtree.h declares,
and rejects invalid arguments on the host with the documented status codes
(no kernel is launched; these run without a GPU)."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2609_33133_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "augtree.h")


def declared_symbols():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(augtree_[a-z_0-9]+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    return _lib.load()


def test_header_declares_the_six_operations():
    syms = declared_symbols()
    for s in ("augtree_prefill_fwd", "augtree_prefill_bwd", "augtree_replay_fwd", "augtree_replay_bwd",
              "augtree_lse_merge", "augtree_prompt_grad_reduce"):
        assert s in syms


def test_every_declared_symbol_is_exported(L):
    for s in declared_symbols():
        assert hasattr(L, s), s
    assert set(declared_symbols()) == set(_lib.EXPORTS)


def test_status_strings(L):
    for code in range(7):
        assert L.augtree_status_string(code).decode() not in ("", "unknown status")
    assert L.augtree_status_string(99).decode() == "unknown status"
    assert L.augtree_version().decode().startswith("augtree")


def groups(cp, cb, cr, hq=4, hkv=2, d=64, scale=0.125):
    cp = np.ascontiguousarray(cp, np.int32)
    cb = np.ascontiguousarray(cb, np.int32)
    cr = np.ascontiguousarray(cr, np.int32)
    p = ctypes.POINTER(ctypes.c_int32)
    g = _lib.Groups(len(cp) - 1, len(cr) - 1, hq, hkv, d, scale, cp.ctypes.data_as(p), cb.ctypes.data_as(p),
                    cr.ctypes.data_as(p))
    g._keep = (cp, cb, cr)
    return g


GOOD = ([0, 10, 25], [0, 2, 3], [0, 5, 12, 20])


def fake(n=1 << 20):
    """A 256-byte-aligned fake device address (never dereferenced: every call
    below fails validation or the device check before any launch)."""
    return ctypes.c_void_p(n * 256)


def test_workspace_size_valid_and_monotone(L):
    g = groups(*GOOD)
    sizes = [L.augtree_workspace_size(ctypes.byref(g), op, 1) for op in range(4)]
    assert all(s > 0 and s % 256 == 0 for s in sizes)
    s1 = L.augtree_workspace_size(ctypes.byref(g), 3, 1)
    s8 = L.augtree_workspace_size(ctypes.byref(g), 3, 8)
    assert s8 >= s1
    big = groups([0, 1000, 2500], [0, 2, 3], [0, 500, 1200, 2000])
    assert L.augtree_workspace_size(ctypes.byref(big), 3, 1) > s1


@pytest.mark.parametrize("cp,cb,cr,hq,hkv,d,code", [
    ([0, 10, 10], [0, 2, 3], [0, 5, 12, 20], 4, 2, 64, 1),   # empty prompt
    ([0, 10, 25], [0, 2, 2], [0, 5, 12, 20], 4, 2, 64, 1),   # group without branch
    ([0, 10, 25], [0, 2, 3], [0, 5, 5, 20], 4, 2, 64, 1),    # empty branch
    ([1, 10, 25], [0, 2, 3], [0, 5, 12, 20], 4, 2, 64, 1),   # offsets not from 0
    ([0, 10, 25], [0, 2, 3], [0, 5, 12, 20], 4, 3, 64, 2),   # Hq % Hkv
    ([0, 10, 25], [0, 2, 3], [0, 5, 12, 20], 4, 2, 96, 2),   # head_dim
])
def test_invalid_descriptors(L, cp, cb, cr, hq, hkv, d, code):
    g = groups(cp, cb, cr, hq, hkv, d)
    assert L.augtree_workspace_size(ctypes.byref(g), 3, 1) == 0
    p = fake()
    st = L.augtree_replay_fwd(ctypes.byref(g), 0, p, p, p, p, p, p, p, None, None, p, 1 << 30, None)
    assert st == code, L.augtree_last_error()
    assert L.augtree_last_error().decode() != ""


def test_null_descriptor_and_pointers(L):
    assert L.augtree_prefill_fwd(None, None, None, None, None, None, None, 0, None) == 1
    g = groups(*GOOD)
    p = fake()
    assert L.augtree_prefill_fwd(ctypes.byref(g), None, p, p, p, p, p, 1 << 30, None) == 1
    assert L.augtree_prefill_fwd(ctypes.byref(g), ctypes.c_void_p(256 * 1000 + 2), p, p, p, p, p, 1 << 30,
                                 None) == 3
    # split mode needs its partial buffers
    assert L.augtree_replay_fwd(ctypes.byref(g), 1, p, p, p, p, p, p, p, None, None, p, 1 << 30, None) == 1
    assert L.augtree_replay_fwd(ctypes.byref(g), 7, p, p, p, p, p, p, p, None, None, p, 1 << 30, None) == 1
    # n_seed range
    assert L.augtree_replay_bwd(ctypes.byref(g), p, p, p, p, p, p, p, p, p, p, p, 0, p, p, 1 << 30, None) == 1
    assert L.augtree_replay_bwd(ctypes.byref(g), p, p, p, p, p, p, p, p, p, p, p, 65, p, p, 1 << 30, None) == 1
    # prefill bwd needs at least one dQ output
    assert L.augtree_prefill_bwd(ctypes.byref(g), p, p, p, p, p, p, None, None, p, p, 1 << 30, None) == 1


def test_prefill_reads_prompt_offsets_only(L):
    cp = np.array([0, 7, 19], np.int32)
    ip = ctypes.POINTER(ctypes.c_int32)
    g = _lib.Groups(2, 0, 4, 4, 64, 0.125, cp.ctypes.data_as(ip), None, None)
    assert L.augtree_workspace_size(ctypes.byref(g), 0, 0) > 0
    assert L.augtree_workspace_size(ctypes.byref(g), 2, 0) > 0
    assert L.augtree_workspace_size(ctypes.byref(g), 1, 0) == 0     # replay needs branches


def test_workspace_checks(L):
    g = groups(*GOOD)
    p = fake()
    need = L.augtree_workspace_size(ctypes.byref(g), 0, 0)
    assert L.augtree_prefill_fwd(ctypes.byref(g), p, p, p, p, p, None, need, None) == 4
    assert L.augtree_prefill_fwd(ctypes.byref(g), p, p, p, p, p, p, need - 1, None) == 4
    assert L.augtree_prefill_fwd(ctypes.byref(g), p, p, p, p, p, ctypes.c_void_p(256 * 1000 + 16), need,
                                 None) == 3


def test_elementwise_argument_checks(L):
    p = fake()
    assert L.augtree_lse_merge(10, 2, 60, 2, p, p, p, None, p, None) == 1        # head_dim % 8
    assert L.augtree_lse_merge(10, 2, 64, 0, p, p, p, None, p, None) == 1        # n_parts
    assert L.augtree_lse_merge(10, 2, 64, 2, p, p, None, None, p, None) == 1     # no output
    assert L.augtree_lse_merge(0, 2, 64, 2, None, None, None, None, None, None) == 0   # empty is a no-op
    assert L.augtree_prompt_grad_reduce(3, 10, 2, 64, None, 1, 10, 0, p, None, p, None, None) == 1
    assert L.augtree_prompt_grad_reduce(2, 10, 2, 64, None, 1, 9, 0, p, None, p, None, None) == 1
    assert L.augtree_prompt_grad_reduce(2, 10, 2, 64, None, 1, 10, 6, p, None, p, None, None) == 1
    assert L.augtree_prompt_grad_reduce(2, 10, 2, 64, None, 1, 10, 0, p, None, None, None, None) == 1


def test_valid_call_without_gpu_reports_device(L):
    """With every argument valid, a host without a gfx950 device gets
    AUGTREE_ERR_DEVICE before anything is enqueued."""
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    g = groups(*GOOD)
    p = fake()
    need = L.augtree_workspace_size(ctypes.byref(g), 0, 0)
    assert L.augtree_prefill_fwd(ctypes.byref(g), p, p, p, p, p, p, need, None) == 5
    assert L.augtree_check_device() == 5


def test_tree_calls_validate_on_the_host(L):
    """The two tree calls reject bad arguments before any launch (statuses as
    for the six calls), and the allocation-free backward rejects a batch whose
    workspace exceeds its fixed device array before touching the device."""
    g = groups(*GOOD)
    p = fake()
    need_f = L.augtree_workspace_size(ctypes.byref(g), 4, 0)
    need_b = L.augtree_workspace_size(ctypes.byref(g), 5, 0)
    assert need_f > 0 and need_b > 0 and need_b % 256 == 0
    assert L.augtree_workspace_size(ctypes.byref(g), 4, 9) == 0          # unknown replay mode
    assert L.augtree_tree_fwd(ctypes.byref(g), 1, *([p] * 6), *([p] * 4), None, None, p, need_f, None) == 1
    assert L.augtree_tree_bwd(ctypes.byref(g), *([p] * 15), None, p, p, None, p, need_b, None) == 1   # null dv_r
    assert L.augtree_tree_bwd(ctypes.byref(g), *([p] * 15), None, p, p, p, p, need_b - 1, None) == 4
    assert L.augtree_noalloc_scratch_bytes() == 64 << 20
    big = groups([0, 1 << 19], [0, 1], [0, 1 << 19], hq=32, hkv=8, d=128)
    assert L.augtree_workspace_size(ctypes.byref(big), 5, 0) > (64 << 20)
    st = L.augtree_tree_bwd_noalloc(ctypes.byref(big), *([p] * 15), None, p, p, p, None)
    assert st == 4 and "allocation-free" in L.augtree_last_error().decode()
