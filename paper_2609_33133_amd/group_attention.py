"""One pass of shared-prompt group attention, forward and backward, on the GPU,
and the flattened per-branch baseline built from the same kernels.

SharedStep (the method, §3.2-§3.3): the prompt prefilled once per tree, every
branch replayed against the prompt KV (read in place) plus its own causal KV, the
branch gradients with every branch's prompt-KV gradient accumulated on the
prompt KV (Eq. 2) together with the prompt queries' own contribution. By
default as augtree_tree_fwd + augtree_tree_bwd; ``path="calls"`` strings the
six separate entry points (prefill_fwd, replay_fwd, replay_bwd, prefill_bwd,
prompt_grad_reduce).

FlattenedStep (the baseline the paper compares against, §2.1): each branch as
its own causal sequence [P; R_i]; the prompt is recomputed once per branch and
the G copies of every prompt gradient are summed afterwards.

Buffers are allocated once per step object (torch), so ``run`` only enqueues
kernels on the current stream.
"""
from __future__ import annotations

import math
from typing import Dict, Optional

import numpy as np
import torch

from . import api
from .api import REPLAY_AUTO, REPLAY_FUSED, REPLAY_SPLIT, GroupBatch

TENSORS = ("q_p", "k_p", "v_p", "q_r", "k_r", "v_r", "do_p", "do_r")


def bf16_tensor(bits: np.ndarray, device) -> torch.Tensor:
    """uint16 bf16 bit patterns (numpy) -> torch.bfloat16 tensor on `device`."""
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(device).view(torch.bfloat16)


def upload(gi, device="cuda") -> Dict[str, torch.Tensor]:
    return {n: bf16_tensor(getattr(gi, n), device) for n in TENSORS}


def default_n_seed(batch: GroupBatch, min_workgroups: int = 1024) -> int:
    """Chunks of the response rows for the prompt-key gradient, so that the
    prompt-key launch has enough workgroups (prompt key tiles x KV heads x
    chunks) to fill the GPU."""
    tiles = sum(math.ceil((batch.cu_prompt[g + 1] - batch.cu_prompt[g]) / 128) for g in range(batch.num_groups))
    work = tiles * batch.hkv
    n = max(1, math.ceil(min_workgroups / max(work, 1)))
    max_rows = max(int(batch.cu_resp[batch.cu_branch[g + 1]] - batch.cu_resp[batch.cu_branch[g]])
                   for g in range(batch.num_groups))
    return int(max(1, min(n, 64, max_rows // 64 if max_rows >= 64 else 1)))


class SharedStep:
    """One step of the method on a fixed batch. ``path="tree"`` (default) runs
    it as augtree_tree_fwd + augtree_tree_bwd (fewest launches; the Eq. 2 sum
    in registers); ``path="calls"`` runs the six separate entry points
    (prefill_fwd, replay_fwd, replay_bwd, prefill_bwd, prompt_grad_reduce)."""

    def __init__(self, batch: GroupBatch, device="cuda", mode: int = REPLAY_FUSED, n_seed: Optional[int] = None,
                 path: str = "tree"):
        if path not in ("tree", "calls"):
            raise ValueError(f"path {path!r}")
        self.b = b = batch
        self.mode = mode
        self.path = path
        self.n_seed = default_n_seed(b) if n_seed is None else int(n_seed)
        dev = torch.device(device)
        f32, bf = torch.float32, torch.bfloat16
        self.o_p = torch.empty((b.tp, b.hq, b.d), dtype=bf, device=dev)
        self.lse_p = torch.empty((b.hq, b.tp), dtype=f32, device=dev)
        self.o_r = torch.empty((b.tr, b.hq, b.d), dtype=bf, device=dev)
        self.lse_r = torch.empty((b.hq, b.tr), dtype=f32, device=dev)
        self.o_part = self.lse_part = None
        if mode != REPLAY_FUSED:
            self.o_part = torch.empty((2, b.tr, b.hq, b.d), dtype=f32, device=dev)
            self.lse_part = torch.empty((2, b.hq, b.tr), dtype=f32, device=dev)
        self.dq_r = torch.empty((b.tr, b.hq, b.d), dtype=bf, device=dev)
        self.dk_r = torch.empty((b.tr, b.hkv, b.d), dtype=bf, device=dev)
        self.dv_r = torch.empty((b.tr, b.hkv, b.d), dtype=bf, device=dev)
        self.dq_p = torch.empty((b.tp, b.hq, b.d), dtype=bf, device=dev)
        self.dkv_p = torch.empty((2, b.tp, b.hkv, b.d), dtype=bf, device=dev)
        if path == "calls":
            self.seed = torch.empty((self.n_seed, 2, b.tp, b.hkv, b.d), dtype=f32, device=dev)
            self.dkv_self = torch.empty((2, b.tp, b.hkv, b.d), dtype=f32, device=dev)
            self.ws = {
                "pf": b.workspace(api.OP_PREFILL_FWD, 0, dev),
                "rf": b.workspace(api.OP_REPLAY_FWD, mode, dev),
                "rb": b.workspace(api.OP_REPLAY_BWD, self.n_seed, dev),
                "pb": b.workspace(api.OP_PREFILL_BWD, 0, dev),
            }
        else:
            self.ws = {"tf": b.workspace(api.OP_TREE_FWD, mode, dev), "tb": b.workspace(api.OP_TREE_BWD, 0, dev)}
        self._bound = None

    def _bind(self, x: Dict[str, torch.Tensor]):
        """ctypes argument tuples of the two tree calls for inputs ``x`` (the
        pointers of every buffer are fixed), so a step is two foreign calls."""
        b, P = self.b, api._ptr
        for n in TENSORS:
            rows = b.tp if n.endswith("_p") else b.tr
            heads = b.hkv if n[0] in "kv" else b.hq
            api._need(x[n], n, torch.bfloat16, (rows, heads, b.d))
        fwd = [b.ref, self.mode, P(x["q_p"]), P(x["k_p"]), P(x["v_p"]), P(x["q_r"]), P(x["k_r"]), P(x["v_r"]),
               P(self.o_p), P(self.lse_p), P(self.o_r), P(self.lse_r), P(self.o_part), P(self.lse_part),
               P(self.ws["tf"]), self.ws["tf"].numel()]
        bwd = [b.ref, P(x["q_p"]), P(x["k_p"]), P(x["v_p"]), P(self.o_p), P(self.lse_p), P(x["do_p"]),
               P(x["q_r"]), P(x["k_r"]), P(x["v_r"]), P(self.o_r), P(self.lse_r), P(x["do_r"]),
               P(self.dq_p), P(self.dkv_p[0]), P(self.dkv_p[1]), None, P(self.dq_r), P(self.dk_r), P(self.dv_r),
               P(self.ws["tb"]), self.ws["tb"].numel()]
        self._bound = (x, fwd, bwd)

    def forward(self, x: Dict[str, torch.Tensor], stream=None):
        b = self.b
        if self.path == "tree":
            if self._bound is None or self._bound[0] is not x:
                self._bind(x)
            lib = api._lib.load()
            api._lib.check(lib.augtree_tree_fwd(*self._bound[1], api._stream(stream)), "tree_fwd")
            return
        api.prefill_fwd(b, x["q_p"], x["k_p"], x["v_p"], self.o_p, self.lse_p, ws=self.ws["pf"], stream=stream)
        api.replay_fwd(b, x["q_r"], x["k_r"], x["v_r"], x["k_p"], x["v_p"], self.mode, self.o_r, self.lse_r,
                       self.o_part, self.lse_part, ws=self.ws["rf"], stream=stream)

    def backward(self, x: Dict[str, torch.Tensor], stream=None):
        b = self.b
        if self.path == "tree":
            if self._bound is None or self._bound[0] is not x:
                self._bind(x)
            lib = api._lib.load()
            api._lib.check(lib.augtree_tree_bwd(*self._bound[2], api._stream(stream)), "tree_bwd")
            return
        api.replay_bwd(b, x["q_r"], x["k_r"], x["v_r"], x["k_p"], x["v_p"], self.o_r, self.lse_r, x["do_r"],
                       self.n_seed, self.dq_r, self.dk_r, self.dv_r, self.seed, ws=self.ws["rb"], stream=stream)
        api.prefill_bwd(b, x["q_p"], x["k_p"], x["v_p"], self.o_p, self.lse_p, x["do_p"], self.dq_p, None,
                        self.dkv_self, ws=self.ws["pb"], stream=stream)
        api.prompt_grad_reduce(self.seed, self_part=self.dkv_self, out=self.dkv_p, stream=stream)

    def run(self, x: Dict[str, torch.Tensor], stream=None):
        self.forward(x, stream)
        self.backward(x, stream)

    def outputs(self) -> Dict[str, torch.Tensor]:
        return {"o_p": self.o_p, "lse_p": self.lse_p, "o_r": self.o_r, "lse_r": self.lse_r,
                "dq_p": self.dq_p, "dk_p": self.dkv_p[0], "dv_p": self.dkv_p[1],
                "dq_r": self.dq_r, "dk_r": self.dk_r, "dv_r": self.dv_r}


class FlattenedStep:
    """Flattened baseline: sequence (g, i) = [P_g; R_i], causal over its
    P_g + R_i rows, prompt rows receiving dO_P / G_g (exact in bf16: G is a
    power of two in every workload here). Prompt gradients of the copies are
    summed with prompt_grad_reduce through row maps."""

    def __init__(self, batch: GroupBatch, device="cuda"):
        self.b = b = batch
        dev = torch.device(device)
        self.dev = dev
        lens, p_src, p_dst, r_src, r_dst, wts = [], [], [], [], [], []
        gmax = max(int(b.cu_branch[g + 1] - b.cu_branch[g]) for g in range(b.num_groups))
        row_map = np.full((gmax, b.tp), -1, dtype=np.int32)
        row = 0
        for g in range(b.num_groups):
            p0, p1 = int(b.cu_prompt[g]), int(b.cu_prompt[g + 1])
            G = int(b.cu_branch[g + 1] - b.cu_branch[g])
            for i, br in enumerate(range(int(b.cu_branch[g]), int(b.cu_branch[g + 1]))):
                r0, r1 = int(b.cu_resp[br]), int(b.cu_resp[br + 1])
                P, R = p1 - p0, r1 - r0
                p_src.append(np.arange(p0, p1)); p_dst.append(np.arange(row, row + P))
                r_src.append(np.arange(r0, r1)); r_dst.append(np.arange(row + P, row + P + R))
                wts.append(np.full(P, 1.0 / G))
                row_map[i, p0:p1] = np.arange(row, row + P)
                lens.append(P + R)
                row += P + R
        self.tf = row
        self.n_parts = gmax
        cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
        self.fb = GroupBatch(cu, np.arange(len(lens) + 1), np.arange(len(lens) + 1), b.hq, b.hkv, b.d, b.scale)
        self.p_src = torch.from_numpy(np.concatenate(p_src)).to(dev)
        self.p_dst = torch.from_numpy(np.concatenate(p_dst)).to(dev)
        self.r_src = torch.from_numpy(np.concatenate(r_src)).to(dev)
        self.r_dst = torch.from_numpy(np.concatenate(r_dst)).to(dev)
        self.p_wt = torch.from_numpy(np.concatenate(wts).astype(np.float32)).to(dev)
        self.row_map = torch.from_numpy(row_map).to(dev)
        f32, bf = torch.float32, torch.bfloat16
        tf = self.tf
        self.x = {n: torch.empty((tf, b.hq if n in ("q", "do") else b.hkv, b.d), dtype=bf, device=dev)
                  for n in ("q", "k", "v", "do")}
        self.o = torch.empty((tf, b.hq, b.d), dtype=bf, device=dev)
        self.lse = torch.empty((b.hq, tf), dtype=f32, device=dev)
        self.dq32 = torch.empty((tf, b.hq, b.d), dtype=f32, device=dev)
        self.dkv = torch.empty((2, tf, b.hkv, b.d), dtype=f32, device=dev)
        self.dq_p = torch.empty((1, b.tp, b.hq, b.d), dtype=bf, device=dev)
        self.dkv_p = torch.empty((2, b.tp, b.hkv, b.d), dtype=bf, device=dev)
        self.ws_f = self.fb.workspace(api.OP_PREFILL_FWD, 0, dev)
        self.ws_b = self.fb.workspace(api.OP_PREFILL_BWD, 0, dev)

    def materialize(self, x: Dict[str, torch.Tensor]):
        """Builds the G private copies (input preparation, not part of a step)."""
        for name, hp, hr in (("q", "q_p", "q_r"), ("k", "k_p", "k_r"), ("v", "v_p", "v_r"), ("do", "do_p", "do_r")):
            t = self.x[name]
            src_p = x[hp].index_select(0, self.p_src)
            if name == "do":
                src_p = (src_p.float() * self.p_wt[:, None, None]).to(torch.bfloat16)
            t.index_copy_(0, self.p_dst, src_p)
            t.index_copy_(0, self.r_dst, x[hr].index_select(0, self.r_src))

    def run(self, stream=None):
        fb, x = self.fb, self.x
        api.prefill_fwd(fb, x["q"], x["k"], x["v"], self.o, self.lse, ws=self.ws_f, stream=stream)
        api.prefill_bwd(fb, x["q"], x["k"], x["v"], self.o, self.lse, x["do"], None, self.dq32, self.dkv,
                        ws=self.ws_b, stream=stream)
        api.prompt_grad_reduce(self.dkv, row_map=self.row_map, rows=self.b.tp, out=self.dkv_p, shared_slab=True,
                               n_parts=self.n_parts, stream=stream)
        api.prompt_grad_reduce(self.dq32[None], row_map=self.row_map, rows=self.b.tp, out=self.dq_p,
                               shared_slab=True, n_parts=self.n_parts, stream=stream)

    def outputs(self) -> Dict[str, torch.Tensor]:
        """Per-tensor results in the shared layout (gathers; for comparison only)."""
        first = self.row_map[0].long()
        return {"o_p": self.o.index_select(0, first), "lse_p": self.lse.index_select(1, first),
                "o_r": self.o.index_select(0, self.r_dst), "lse_r": self.lse.index_select(1, self.r_dst),
                "dq_p": self.dq_p[0], "dk_p": self.dkv_p[0], "dv_p": self.dkv_p[1],
                "dq_r": self.dq32.index_select(0, self.r_dst).to(torch.bfloat16),
                "dk_r": self.dkv[0].index_select(0, self.r_dst).to(torch.bfloat16),
                "dv_r": self.dkv[1].index_select(0, self.r_dst).to(torch.bfloat16)}
