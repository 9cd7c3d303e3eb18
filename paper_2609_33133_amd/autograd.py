"""Shared-prompt group attention as a differentiable torch op on one GPU.

    o_p, o_r = group_attention(q_p, k_p, v_p, q_r, k_r, v_r, batch)

Inputs are the packed bf16 tensors of a batch of replay trees (prompt rows
[T_P, H, d], response rows [T_R, H, d], `batch` the GroupBatch holding their
offsets). Forward: augtree_tree_fwd (the prompt, causal, once per tree, and
every branch against the prompt KV, read in place, plus its own causal KV; §3.2,
Eq. 1). Backward: augtree_tree_bwd (branch gradients, and the prompt-KV
gradient of every branch plus the prompt queries' own contribution summed on
the prompt KV in a fixed order, Eq. 2). Every step runs in the library's
kernels on the current stream; autograd only routes tensors. There is no CPU
path.
"""
from __future__ import annotations

from typing import Tuple

import torch

from . import api
from .api import REPLAY_FUSED, GroupBatch


def _check(t: torch.Tensor, name: str, rows: int, heads: int, d: int):
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a GPU tensor (the op has no CPU path)")
    if t.dtype != torch.bfloat16:
        raise TypeError(f"{name}: dtype {t.dtype}, expected torch.bfloat16")
    if tuple(t.shape) != (rows, heads, d):
        raise ValueError(f"{name}: shape {tuple(t.shape)}, expected {(rows, heads, d)}")


class _GroupAttention(torch.autograd.Function):
    @staticmethod
    def forward(ctx, q_p, k_p, v_p, q_r, k_r, v_r, batch: GroupBatch, mode: int):
        b = batch
        for t, n, rows, h in ((q_p, "q_p", b.tp, b.hq), (k_p, "k_p", b.tp, b.hkv), (v_p, "v_p", b.tp, b.hkv),
                              (q_r, "q_r", b.tr, b.hq), (k_r, "k_r", b.tr, b.hkv), (v_r, "v_r", b.tr, b.hkv)):
            _check(t, n, rows, h, b.d)
        q_p, k_p, v_p, q_r, k_r, v_r = (t.contiguous() for t in (q_p, k_p, v_p, q_r, k_r, v_r))
        o_p, lse_p, o_r, lse_r = api.tree_fwd(b, q_p, k_p, v_p, q_r, k_r, v_r, mode)[:4]
        ctx.save_for_backward(q_p, k_p, v_p, q_r, k_r, v_r, o_p, lse_p, o_r, lse_r)
        ctx.batch = b
        ctx.mark_non_differentiable(lse_p, lse_r)
        return o_p, o_r

    @staticmethod
    def backward(ctx, do_p, do_r):
        b = ctx.batch
        q_p, k_p, v_p, q_r, k_r, v_r, o_p, lse_p, o_r, lse_r = ctx.saved_tensors
        # an output that did not reach the loss has a zero gradient
        do_p = torch.zeros_like(o_p) if do_p is None else do_p.to(torch.bfloat16).contiguous()
        do_r = torch.zeros_like(o_r) if do_r is None else do_r.to(torch.bfloat16).contiguous()
        dq_p, dk_p, dv_p, dq_r, dk_r, dv_r, _ = api.tree_bwd(b, q_p, k_p, v_p, o_p, lse_p, do_p, q_r, k_r, v_r, o_r,
                                                             lse_r, do_r)
        return dq_p, dk_p, dv_p, dq_r, dk_r, dv_r, None, None


def group_attention(q_p: torch.Tensor, k_p: torch.Tensor, v_p: torch.Tensor, q_r: torch.Tensor,
                    k_r: torch.Tensor, v_r: torch.Tensor, batch: GroupBatch,
                    mode: int = REPLAY_FUSED) -> Tuple[torch.Tensor, torch.Tensor]:
    """(O_P, O_R) of shared-prompt group attention; differentiable in all six inputs."""
    return _GroupAttention.apply(q_p, k_p, v_p, q_r, k_r, v_r, batch, int(mode))
