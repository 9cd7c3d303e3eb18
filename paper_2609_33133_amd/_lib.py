"""ctypes loader of libaugtree.so (the C ABI declared in include/augtree.h).

torch is imported before the library is opened: torch ships its own HIP
runtime with the same SONAME (libamdhip64.so.7), so the library binds to that
copy and shares torch's devices, memory and streams. A missing library is an
error; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libaugtree.so")

AUGTREE_OK = 0
AUGTREE_ERR_INVALID_ARGUMENT = 1
AUGTREE_ERR_UNSUPPORTED = 2
AUGTREE_ERR_MISALIGNED = 3
AUGTREE_ERR_WORKSPACE = 4
AUGTREE_ERR_DEVICE = 5
AUGTREE_ERR_HIP = 6

REPLAY_FUSED = 0
REPLAY_SPLIT = 1
REPLAY_AUTO = 2

OP_PREFILL_FWD = 0
OP_REPLAY_FWD = 1
OP_PREFILL_BWD = 2
OP_REPLAY_BWD = 3
OP_TREE_FWD = 4
OP_TREE_BWD = 5

EXPORTS = (
    "augtree_workspace_size", "augtree_prefill_fwd", "augtree_replay_fwd", "augtree_lse_merge",
    "augtree_replay_bwd", "augtree_prefill_bwd", "augtree_prompt_grad_reduce", "augtree_status_string",
    "augtree_last_error", "augtree_check_device", "augtree_version", "augtree_set_launch_hook",
    "augtree_replay_split_groups", "augtree_tree_fwd", "augtree_tree_bwd", "augtree_tree_bwd_noalloc",
    "augtree_noalloc_scratch_bytes", "augtree_set_tree_chunk_blocks", "augtree_tree_chunk_blocks",
)

LAUNCH_HOOK = ctypes.CFUNCTYPE(None, ctypes.c_char_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p)


class Groups(ctypes.Structure):
    """struct augtree_groups."""
    _fields_ = [
        ("num_groups", ctypes.c_int32),
        ("num_branches", ctypes.c_int32),
        ("num_q_heads", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("softmax_scale", ctypes.c_float),
        ("cu_prompt", ctypes.POINTER(ctypes.c_int32)),
        ("cu_branch", ctypes.POINTER(ctypes.c_int32)),
        ("cu_resp", ctypes.POINTER(ctypes.c_int32)),
    ]


class AugtreeError(RuntimeError):
    def __init__(self, status: int, what: str, detail: str):
        super().__init__(f"{what}: status {status}: {detail}")
        self.status = status


_lib = None

_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_I64 = ctypes.c_int64
_SZ = ctypes.c_size_t
_GP = ctypes.POINTER(Groups)


def _sig(lib):
    sigs = {
        "augtree_workspace_size": (_SZ, [_GP, ctypes.c_int, ctypes.c_int]),
        "augtree_prefill_fwd": (ctypes.c_int, [_GP, _P, _P, _P, _P, _P, _P, _SZ, _P]),
        "augtree_replay_fwd": (ctypes.c_int, [_GP, ctypes.c_int, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
        "augtree_lse_merge": (ctypes.c_int, [_I64, _I32, _I32, _I32, _P, _P, _P, _P, _P, _P]),
        "augtree_replay_bwd": (ctypes.c_int, [_GP, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _I32, _P, _P, _SZ, _P]),
        "augtree_prefill_bwd": (ctypes.c_int, [_GP, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
        "augtree_prompt_grad_reduce": (ctypes.c_int, [_I32, _I64, _I32, _I32, _P, _I32, _I64, _I64, _P, _P, _P, _P, _P]),
        "augtree_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "augtree_last_error": (ctypes.c_char_p, []),
        "augtree_check_device": (ctypes.c_int, []),
        "augtree_version": (ctypes.c_char_p, []),
        "augtree_set_launch_hook": (None, [LAUNCH_HOOK, ctypes.c_void_p]),
        "augtree_replay_split_groups": (ctypes.c_int, [_GP, _P]),
        "augtree_tree_fwd": (ctypes.c_int, [_GP, ctypes.c_int] + [_P] * 12 + [_P, _SZ, _P]),
        "augtree_tree_bwd": (ctypes.c_int, [_GP] + [_P] * 19 + [_P, _SZ, _P]),
        "augtree_tree_bwd_noalloc": (ctypes.c_int, [_GP] + [_P] * 19 + [_P]),
        "augtree_noalloc_scratch_bytes": (_SZ, []),
        "augtree_set_tree_chunk_blocks": (ctypes.c_int, [_I32]),
        "augtree_tree_chunk_blocks": (_I32, []),
    }
    for name, (res, args) in sigs.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args


def load(path: str = LIB_PATH):
    """Open libaugtree.so once (after torch) and declare its signatures."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"libaugtree.so not built at {path}; run python -m paper_2609_33133_amd.build")
    import torch  # noqa: F401  (binds the library to torch's HIP runtime)
    lib = ctypes.CDLL(path)
    _sig(lib)
    _lib = lib
    return lib


def check(status: int, what: str):
    if status != AUGTREE_OK:
        lib = load()
        raise AugtreeError(status, what, lib.augtree_last_error().decode())
