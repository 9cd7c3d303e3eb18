"""Thin Python binding over the C ABI (include/augtree.h).

Argument marshalling only: every step of the computation runs in the HIP
kernels of libaugtree.so. torch provides device memory (outputs and
workspace are allocated with torch when the caller passes none) and the
current HIP stream. Function names and argument order follow the C entry
points without the ``augtree_`` prefix.
"""
from __future__ import annotations

import ctypes
import math
from typing import Optional, Sequence

import numpy as np
import torch

from . import _lib
from ._lib import (REPLAY_FUSED, REPLAY_SPLIT, REPLAY_AUTO, OP_PREFILL_FWD, OP_REPLAY_FWD,  # noqa: F401
                   OP_PREFILL_BWD, OP_REPLAY_BWD, OP_TREE_FWD, OP_TREE_BWD)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _need(t: torch.Tensor, name: str, dtype, shape):
    if t.dtype != dtype:
        raise TypeError(f"{name}: dtype {t.dtype}, expected {dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: shape {tuple(t.shape)}, expected {tuple(shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a device tensor")


class GroupBatch:
    """A batch of replay trees (struct augtree_groups) with its host offsets."""

    def __init__(self, cu_prompt, cu_branch, cu_resp, num_q_heads: int, num_kv_heads: int, head_dim: int,
                 softmax_scale: Optional[float] = None):
        self.cu_prompt = np.ascontiguousarray(cu_prompt, dtype=np.int32)
        self.cu_branch = np.ascontiguousarray(cu_branch, dtype=np.int32)
        self.cu_resp = np.ascontiguousarray(cu_resp, dtype=np.int32)
        self.num_groups = len(self.cu_prompt) - 1
        self.num_branches = len(self.cu_resp) - 1
        self.hq, self.hkv, self.d = int(num_q_heads), int(num_kv_heads), int(head_dim)
        self.scale = float(softmax_scale if softmax_scale is not None else 1.0 / math.sqrt(head_dim))
        self.tp = int(self.cu_prompt[-1])
        self.tr = int(self.cu_resp[-1])
        i32p = ctypes.POINTER(ctypes.c_int32)
        self.struct = _lib.Groups(self.num_groups, self.num_branches, self.hq, self.hkv, self.d, self.scale,
                                  self.cu_prompt.ctypes.data_as(i32p), self.cu_branch.ctypes.data_as(i32p),
                                  self.cu_resp.ctypes.data_as(i32p))

    @classmethod
    def from_shape(cls, shape) -> "GroupBatch":
        return cls(shape.cu_prompt, shape.cu_branch, shape.cu_resp, shape.num_q_heads, shape.num_kv_heads,
                   shape.head_dim, shape.scale)

    @property
    def ref(self):
        return ctypes.byref(self.struct)

    def workspace_size(self, op: int, arg: int = 0) -> int:
        lib = _lib.load()
        n = lib.augtree_workspace_size(self.ref, op, arg)
        if n == 0:
            raise _lib.AugtreeError(_lib.AUGTREE_ERR_INVALID_ARGUMENT, "workspace_size",
                                    lib.augtree_last_error().decode())
        return int(n)

    def workspace(self, op: int, arg: int = 0, device=None) -> torch.Tensor:
        return torch.empty(self.workspace_size(op, arg), dtype=torch.uint8, device=device or "cuda")


def _ws(b: GroupBatch, ws, op, arg, device):
    if ws is None:
        ws = b.workspace(op, arg, device)
    return ws, ctypes.c_size_t(ws.numel())


def prefill_fwd(b: GroupBatch, q_p, k_p, v_p, o_p=None, lse_p=None, ws=None, stream=None):
    _need(q_p, "q_p", torch.bfloat16, (b.tp, b.hq, b.d))
    _need(k_p, "k_p", torch.bfloat16, (b.tp, b.hkv, b.d))
    _need(v_p, "v_p", torch.bfloat16, (b.tp, b.hkv, b.d))
    o_p = torch.empty_like(q_p) if o_p is None else o_p
    lse_p = torch.empty((b.hq, b.tp), dtype=torch.float32, device=q_p.device) if lse_p is None else lse_p
    _need(o_p, "o_p", torch.bfloat16, q_p.shape)
    _need(lse_p, "lse_p", torch.float32, (b.hq, b.tp))
    ws, nws = _ws(b, ws, OP_PREFILL_FWD, 0, q_p.device)
    _lib.check(_lib.load().augtree_prefill_fwd(b.ref, _ptr(q_p), _ptr(k_p), _ptr(v_p), _ptr(o_p), _ptr(lse_p),
                                               _ptr(ws), nws, _stream(stream)), "prefill_fwd")
    return o_p, lse_p


def replay_fwd(b: GroupBatch, q_r, k_r, v_r, k_p, v_p, mode: int = REPLAY_FUSED, o_r=None, lse_r=None,
               o_part=None, lse_part=None, ws=None, stream=None):
    _need(q_r, "q_r", torch.bfloat16, (b.tr, b.hq, b.d))
    _need(k_r, "k_r", torch.bfloat16, (b.tr, b.hkv, b.d))
    _need(v_r, "v_r", torch.bfloat16, (b.tr, b.hkv, b.d))
    _need(k_p, "k_p", torch.bfloat16, (b.tp, b.hkv, b.d))
    _need(v_p, "v_p", torch.bfloat16, (b.tp, b.hkv, b.d))
    dev = q_r.device
    o_r = torch.empty_like(q_r) if o_r is None else o_r
    lse_r = torch.empty((b.hq, b.tr), dtype=torch.float32, device=dev) if lse_r is None else lse_r
    if mode != REPLAY_FUSED:
        o_part = torch.empty((2, b.tr, b.hq, b.d), dtype=torch.float32, device=dev) if o_part is None else o_part
        lse_part = torch.empty((2, b.hq, b.tr), dtype=torch.float32, device=dev) if lse_part is None else lse_part
    ws, nws = _ws(b, ws, OP_REPLAY_FWD, mode, dev)
    _lib.check(_lib.load().augtree_replay_fwd(b.ref, mode, _ptr(q_r), _ptr(k_r), _ptr(v_r), _ptr(k_p), _ptr(v_p),
                                              _ptr(o_r), _ptr(lse_r), _ptr(o_part), _ptr(lse_part), _ptr(ws), nws,
                                              _stream(stream)), "replay_fwd")
    return o_r, lse_r, o_part, lse_part


def replay_split_groups(b: GroupBatch) -> np.ndarray:
    """Per group, 1 if AUGTREE_REPLAY_AUTO runs it SPLIT, 0 if FUSED."""
    out = np.zeros(b.num_groups, dtype=np.int32)
    _lib.check(_lib.load().augtree_replay_split_groups(b.ref, out.ctypes.data_as(ctypes.c_void_p)),
               "replay_split_groups")
    return out


def set_tree_chunk_blocks(blocks: int) -> None:
    """Most query blocks (64 rows x one query head) a prompt-key tile of the
    tree backward sweeps over a group's branch rows before the sweep is cut
    into chunks (0 restores the default). Process-wide; workspaces sized
    afterwards follow it."""
    _lib.check(_lib.load().augtree_set_tree_chunk_blocks(int(blocks)), "set_tree_chunk_blocks")


def tree_chunk_blocks() -> int:
    return int(_lib.load().augtree_tree_chunk_blocks())


def lse_merge(o_parts, lse_parts, o=None, o_f32=None, lse=None, want_bf16=True, stream=None):
    n, rows, heads, d = o_parts.shape
    _need(o_parts, "o_parts", torch.float32, (n, rows, heads, d))
    _need(lse_parts, "lse_parts", torch.float32, (n, heads, rows))
    dev = o_parts.device
    if o is None and o_f32 is None:
        if want_bf16:
            o = torch.empty((rows, heads, d), dtype=torch.bfloat16, device=dev)
        else:
            o_f32 = torch.empty((rows, heads, d), dtype=torch.float32, device=dev)
    lse = torch.empty((heads, rows), dtype=torch.float32, device=dev) if lse is None else lse
    _lib.check(_lib.load().augtree_lse_merge(rows, heads, d, n, _ptr(o_parts), _ptr(lse_parts), _ptr(o),
                                             _ptr(o_f32), _ptr(lse), _stream(stream)), "lse_merge")
    return o, o_f32, lse


def replay_bwd(b: GroupBatch, q_r, k_r, v_r, k_p, v_p, o_r, lse_r, do_r, n_seed: int = 1, dq_r=None, dk_r=None,
               dv_r=None, dkv_p_seed=None, ws=None, stream=None):
    for t, nm, h in ((q_r, "q_r", b.hq), (o_r, "o_r", b.hq), (do_r, "do_r", b.hq), (k_r, "k_r", b.hkv),
                     (v_r, "v_r", b.hkv)):
        _need(t, nm, torch.bfloat16, (b.tr, h, b.d))
    _need(k_p, "k_p", torch.bfloat16, (b.tp, b.hkv, b.d))
    _need(v_p, "v_p", torch.bfloat16, (b.tp, b.hkv, b.d))
    _need(lse_r, "lse_r", torch.float32, (b.hq, b.tr))
    dev = q_r.device
    dq_r = torch.empty_like(q_r) if dq_r is None else dq_r
    dk_r = torch.empty_like(k_r) if dk_r is None else dk_r
    dv_r = torch.empty_like(v_r) if dv_r is None else dv_r
    if dkv_p_seed is None:
        dkv_p_seed = torch.empty((n_seed, 2, b.tp, b.hkv, b.d), dtype=torch.float32, device=dev)
    _need(dkv_p_seed, "dkv_p_seed", torch.float32, (n_seed, 2, b.tp, b.hkv, b.d))
    ws, nws = _ws(b, ws, OP_REPLAY_BWD, n_seed, dev)
    _lib.check(_lib.load().augtree_replay_bwd(b.ref, _ptr(q_r), _ptr(k_r), _ptr(v_r), _ptr(k_p), _ptr(v_p),
                                              _ptr(o_r), _ptr(lse_r), _ptr(do_r), _ptr(dq_r), _ptr(dk_r),
                                              _ptr(dv_r), n_seed, _ptr(dkv_p_seed), _ptr(ws), nws,
                                              _stream(stream)), "replay_bwd")
    return dq_r, dk_r, dv_r, dkv_p_seed


def prefill_bwd(b: GroupBatch, q_p, k_p, v_p, o_p, lse_p, do_p, dq_p=None, dq_p_f32=None, dkv_p_self=None,
                want_bf16=True, ws=None, stream=None):
    for t, nm, h in ((q_p, "q_p", b.hq), (o_p, "o_p", b.hq), (do_p, "do_p", b.hq), (k_p, "k_p", b.hkv),
                     (v_p, "v_p", b.hkv)):
        _need(t, nm, torch.bfloat16, (b.tp, h, b.d))
    _need(lse_p, "lse_p", torch.float32, (b.hq, b.tp))
    dev = q_p.device
    if dq_p is None and dq_p_f32 is None:
        if want_bf16:
            dq_p = torch.empty_like(q_p)
        else:
            dq_p_f32 = torch.empty(q_p.shape, dtype=torch.float32, device=dev)
    if dkv_p_self is None:
        dkv_p_self = torch.empty((2, b.tp, b.hkv, b.d), dtype=torch.float32, device=dev)
    _need(dkv_p_self, "dkv_p_self", torch.float32, (2, b.tp, b.hkv, b.d))
    ws, nws = _ws(b, ws, OP_PREFILL_BWD, 0, dev)
    _lib.check(_lib.load().augtree_prefill_bwd(b.ref, _ptr(q_p), _ptr(k_p), _ptr(v_p), _ptr(o_p), _ptr(lse_p),
                                               _ptr(do_p), _ptr(dq_p), _ptr(dq_p_f32), _ptr(dkv_p_self), _ptr(ws),
                                               nws, _stream(stream)), "prefill_bwd")
    return dq_p, dq_p_f32, dkv_p_self


def prompt_grad_reduce(parts, self_part=None, row_map=None, rows: Optional[int] = None, out=None, out_f32=None,
                       want_bf16=True, shared_slab: bool = False, n_parts: Optional[int] = None, stream=None):
    """Eq. 2 sum. ``parts`` is [n_parts, n_tensors, part_rows, heads, d] fp32
    (one slab per term), or, with ``shared_slab=True``, a single slab
    [n_tensors, part_rows, heads, d] that every one of the ``n_parts`` terms
    reads through ``row_map`` [n_parts, rows] (int32, -1 = no row).
    Returns (out bf16 [n_tensors, rows, heads, d] or None, out_f32 or None)."""
    if shared_slab:
        n_tensors, part_rows, heads, d = parts.shape
        if row_map is None or n_parts is None:
            raise ValueError("shared_slab needs row_map and n_parts")
        part_stride = 0
    else:
        n_parts, n_tensors, part_rows, heads, d = parts.shape
        part_stride = n_tensors * part_rows * heads * d
    _need(parts, "parts", torch.float32, parts.shape)
    rows = part_rows if rows is None else int(rows)
    if self_part is not None:
        _need(self_part, "self", torch.float32, (n_tensors, rows, heads, d))
    if row_map is not None:
        _need(row_map, "row_map", torch.int32, (n_parts, rows))
    dev = parts.device
    if out is None and out_f32 is None:
        if want_bf16:
            out = torch.empty((n_tensors, rows, heads, d), dtype=torch.bfloat16, device=dev)
        else:
            out_f32 = torch.empty((n_tensors, rows, heads, d), dtype=torch.float32, device=dev)
    _lib.check(_lib.load().augtree_prompt_grad_reduce(n_tensors, rows, heads, d, _ptr(self_part), n_parts, part_rows,
                                                      part_stride, _ptr(parts), _ptr(row_map), _ptr(out),
                                                      _ptr(out_f32), _stream(stream)), "prompt_grad_reduce")
    return out, out_f32


def tree_fwd(b: GroupBatch, q_p, k_p, v_p, q_r, k_r, v_r, mode: int = REPLAY_FUSED, o_p=None, lse_p=None, o_r=None,
             lse_r=None, o_part=None, lse_part=None, ws=None, stream=None):
    """Prefill + replay forward of every tree in one call (augtree_tree_fwd).
    Returns (o_p, lse_p, o_r, lse_r, o_part, lse_part)."""
    for t, nm, rows, h in ((q_p, "q_p", b.tp, b.hq), (k_p, "k_p", b.tp, b.hkv), (v_p, "v_p", b.tp, b.hkv),
                           (q_r, "q_r", b.tr, b.hq), (k_r, "k_r", b.tr, b.hkv), (v_r, "v_r", b.tr, b.hkv)):
        _need(t, nm, torch.bfloat16, (rows, h, b.d))
    dev = q_p.device
    o_p = torch.empty_like(q_p) if o_p is None else o_p
    o_r = torch.empty_like(q_r) if o_r is None else o_r
    lse_p = torch.empty((b.hq, b.tp), dtype=torch.float32, device=dev) if lse_p is None else lse_p
    lse_r = torch.empty((b.hq, b.tr), dtype=torch.float32, device=dev) if lse_r is None else lse_r
    _need(o_p, "o_p", torch.bfloat16, q_p.shape)
    _need(o_r, "o_r", torch.bfloat16, q_r.shape)
    _need(lse_p, "lse_p", torch.float32, (b.hq, b.tp))
    _need(lse_r, "lse_r", torch.float32, (b.hq, b.tr))
    if mode != REPLAY_FUSED:
        o_part = torch.empty((2, b.tr, b.hq, b.d), dtype=torch.float32, device=dev) if o_part is None else o_part
        lse_part = torch.empty((2, b.hq, b.tr), dtype=torch.float32, device=dev) if lse_part is None else lse_part
    ws, nws = _ws(b, ws, OP_TREE_FWD, mode, dev)
    _lib.check(_lib.load().augtree_tree_fwd(b.ref, mode, _ptr(q_p), _ptr(k_p), _ptr(v_p), _ptr(q_r), _ptr(k_r),
                                            _ptr(v_r), _ptr(o_p), _ptr(lse_p), _ptr(o_r), _ptr(lse_r), _ptr(o_part),
                                            _ptr(lse_part), _ptr(ws), nws, _stream(stream)), "tree_fwd")
    return o_p, lse_p, o_r, lse_r, o_part, lse_part


def tree_bwd(b: GroupBatch, q_p, k_p, v_p, o_p, lse_p, do_p, q_r, k_r, v_r, o_r, lse_r, do_r, dq_p=None, dk_p=None,
             dv_p=None, dkv_p_f32=None, dq_r=None, dk_r=None, dv_r=None, want_f32=False, ws=None, stream=None):
    """Gradients of every tree in one call (augtree_tree_bwd): the Eq. 2 sum of
    the prompt-key gradient is formed in registers. Returns
    (dq_p, dk_p, dv_p, dq_r, dk_r, dv_r, dkv_p_f32 or None)."""
    for t, nm, rows, h in ((q_p, "q_p", b.tp, b.hq), (k_p, "k_p", b.tp, b.hkv), (v_p, "v_p", b.tp, b.hkv),
                           (o_p, "o_p", b.tp, b.hq), (do_p, "do_p", b.tp, b.hq),
                           (q_r, "q_r", b.tr, b.hq), (k_r, "k_r", b.tr, b.hkv), (v_r, "v_r", b.tr, b.hkv),
                           (o_r, "o_r", b.tr, b.hq), (do_r, "do_r", b.tr, b.hq)):
        _need(t, nm, torch.bfloat16, (rows, h, b.d))
    _need(lse_p, "lse_p", torch.float32, (b.hq, b.tp))
    _need(lse_r, "lse_r", torch.float32, (b.hq, b.tr))
    dev = q_p.device
    dq_p = torch.empty_like(q_p) if dq_p is None else dq_p
    dk_p = torch.empty_like(k_p) if dk_p is None else dk_p
    dv_p = torch.empty_like(v_p) if dv_p is None else dv_p
    dq_r = torch.empty_like(q_r) if dq_r is None else dq_r
    dk_r = torch.empty_like(k_r) if dk_r is None else dk_r
    dv_r = torch.empty_like(v_r) if dv_r is None else dv_r
    for t, nm, ref in ((dq_p, "dq_p", q_p), (dk_p, "dk_p", k_p), (dv_p, "dv_p", v_p), (dq_r, "dq_r", q_r),
                       (dk_r, "dk_r", k_r), (dv_r, "dv_r", v_r)):
        _need(t, nm, torch.bfloat16, ref.shape)
    if dkv_p_f32 is None and want_f32:
        dkv_p_f32 = torch.empty((2, b.tp, b.hkv, b.d), dtype=torch.float32, device=dev)
    if dkv_p_f32 is not None:
        _need(dkv_p_f32, "dkv_p_f32", torch.float32, (2, b.tp, b.hkv, b.d))
    ws, nws = _ws(b, ws, OP_TREE_BWD, 0, dev)
    _lib.check(_lib.load().augtree_tree_bwd(b.ref, _ptr(q_p), _ptr(k_p), _ptr(v_p), _ptr(o_p), _ptr(lse_p),
                                            _ptr(do_p), _ptr(q_r), _ptr(k_r), _ptr(v_r), _ptr(o_r), _ptr(lse_r),
                                            _ptr(do_r), _ptr(dq_p), _ptr(dk_p), _ptr(dv_p), _ptr(dkv_p_f32),
                                            _ptr(dq_r), _ptr(dk_r), _ptr(dv_r), _ptr(ws), nws, _stream(stream)),
               "tree_bwd")
    return dq_p, dk_p, dv_p, dq_r, dk_r, dv_r, dkv_p_f32
