"""Seeded synthetic inputs for shared-prompt group attention.

This module holds no attention arithmetic. It only draws lengths and tensors,
so that the fp64 oracle (test infrastructure) and the HIP path consume the same
bf16 bit patterns.

Workloads (synthetic stand-ins for the paper's post-training corpora, which are
not available here; §4.1 builds its replay sets from long-context alignment,
chat and reasoning-trace corpora):

* ``tiny``      1 group, P=256, G=2, R=128, Hq=Hkv=4, d=64, seed 0.
* ``balanced``  4 groups, each P=4096, G=8, R=4096, Hq=32, Hkv=8, d=128.
* ``prompt``    1 group, P=32768, G=8, R=2048 (prompt-heavy regime).
* ``response``  1 group, P=2048, G=16, R=16384 (response-heavy regime).
* ``ragged``    16 groups, P log-uniform in [512, 65536], G uniform in
                {4, 8, 16}, every R log-uniform in [256, 32768], packed total
                capped at 1,048,576 tokens, seed 7.

Layout (packed varlen, the layout every entry point takes):
  prompt tensors   Q_P [T_P, Hq, d], K_P/V_P [T_P, Hkv, d]
  response tensors Q_R [T_R, Hq, d], K_R/V_R [T_R, Hkv, d]
  bf16 stored as uint16 bit patterns, head_dim innermost.
Offsets: cu_prompt [num_groups+1] (prompt rows of group g),
cu_branch [num_groups+1] (group g owns branches cu_branch[g]..cu_branch[g+1]),
cu_resp [num_branches+1] (response rows of branch b).

Tensors: Q_P, K_P, V_P, Q_R, K_R, V_R, dO_P, dO_R (tensor index 0..7). Each
packed array is cut into chunks of CHUNK_ROWS rows; chunk c of tensor t is
``standard_normal(float32)`` from its own PCG64 stream seeded with
``SeedSequence([seed, t, c])`` (independent streams, drawn in parallel
threads). Q, K, V are multiplied by 1/sqrt(d) in fp32, dO is not scaled;
fp32 -> bf16 by round-to-nearest-even. The ragged lengths are drawn first from
the main stream ``PCG64(seed)``.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Sequence

import numpy as np

TOKEN_CAP = 1_048_576


@dataclasses.dataclass(frozen=True)
class GroupShape:
    """Lengths of a batch of replay trees plus the attention head shape."""
    prompt_lens: tuple          # P_g per group
    branch_lens: tuple          # tuple of tuples: R_{g,i}
    num_q_heads: int
    num_kv_heads: int
    head_dim: int

    @property
    def num_groups(self) -> int:
        return len(self.prompt_lens)

    @property
    def num_branches(self) -> int:
        return sum(len(r) for r in self.branch_lens)

    @property
    def cu_prompt(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.prompt_lens)]).astype(np.int32)

    @property
    def cu_branch(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum([len(r) for r in self.branch_lens])]).astype(np.int32)

    @property
    def cu_resp(self) -> np.ndarray:
        flat = [x for r in self.branch_lens for x in r]
        return np.concatenate([[0], np.cumsum(flat)]).astype(np.int32)

    @property
    def total_prompt(self) -> int:
        return int(sum(self.prompt_lens))

    @property
    def total_resp(self) -> int:
        return int(sum(sum(r) for r in self.branch_lens))

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.head_dim)

    def valid_pairs(self) -> Dict[str, int]:
        """Query-key pairs with a visible key, per step of the method (integer counts)."""
        prefill = sum(p * (p + 1) // 2 for p in self.prompt_lens)
        rp = sum(p * sum(rs) for p, rs in zip(self.prompt_lens, self.branch_lens))
        rr = sum(r * (r + 1) // 2 for rs in self.branch_lens for r in rs)
        flat = sum((p + r) * (p + r + 1) // 2
                   for p, rs in zip(self.prompt_lens, self.branch_lens) for r in rs)
        return {"prefill": prefill, "replay_prompt": rp, "replay_resp": rr,
                "shared": prefill + rp + rr, "flattened": flat}


def _fixed(P: int, G: int, R: int, groups: int, hq: int, hkv: int, d: int) -> GroupShape:
    return GroupShape(tuple([P] * groups), tuple(tuple([R] * G) for _ in range(groups)), hq, hkv, d)


def ragged_lengths(rng: np.random.Generator, num_groups: int = 16, cap: int = TOKEN_CAP,
                   max_attempts: int = 10_000):
    """Draw the ragged batch: per group P, then G, then each R_i; redraw the whole
    batch from the continuing stream until the packed total fits the cap.
    Returns (prompt_lens, branch_lens, attempts)."""
    lo_p, hi_p = math.log(512.0), math.log(65536.0)
    lo_r, hi_r = math.log(256.0), math.log(32768.0)
    for attempt in range(1, max_attempts + 1):
        ps, rs = [], []
        for _ in range(num_groups):
            p = int(np.round(np.exp(rng.uniform(lo_p, hi_p))))
            g = [4, 8, 16][int(rng.integers(0, 3))]
            r = [int(np.round(np.exp(rng.uniform(lo_r, hi_r)))) for _ in range(g)]
            ps.append(p)
            rs.append(tuple(r))
        if sum(ps) + sum(sum(r) for r in rs) <= cap:
            return tuple(ps), tuple(rs), attempt
    raise RuntimeError("ragged sampler: no batch under the token cap")


CONFIG_NAMES = ("tiny", "balanced", "prompt", "response", "ragged")
# Group-size sweep at a fixed 65,536 response tokens per tree (P = 8192,
# G in {8, 16, 32, 64}, R = 65536 / G) and the prompt-heavy tree with the
# 28 query / 4 KV heads of a 7B model (g = 7, not a power of two), and a
# short-answer tree (P = 16384, G = 32, R = 64) where the replay forward's
# per-group mode rule chooses the split form.
SWEEP_NAMES = ("gsweep8", "gsweep16", "gsweep32", "gsweep64", "prompt_gqa7", "short_resp")
CONFIG_SEEDS = {"tiny": 0, "balanced": 0, "prompt": 0, "response": 0, "ragged": 7,
                **{n: 0 for n in SWEEP_NAMES}}


def config_shape(name: str) -> GroupShape:
    """Shape of a named workload. The ragged shape consumes its seed's stream."""
    if name == "tiny":
        return _fixed(256, 2, 128, 1, 4, 4, 64)
    if name == "balanced":
        return _fixed(4096, 8, 4096, 4, 32, 8, 128)
    if name == "prompt":
        return _fixed(32768, 8, 2048, 1, 32, 8, 128)
    if name == "response":
        return _fixed(2048, 16, 16384, 1, 32, 8, 128)
    if name == "ragged":
        rng = np.random.Generator(np.random.PCG64(CONFIG_SEEDS["ragged"]))
        ps, rs, _ = ragged_lengths(rng)
        return GroupShape(ps, rs, 32, 8, 128)
    if name.startswith("gsweep"):
        g = int(name[len("gsweep"):])
        return _fixed(8192, g, 65536 // g, 1, 32, 8, 128)
    if name == "prompt_gqa7":
        return _fixed(32768, 8, 2048, 1, 28, 4, 128)
    if name == "short_resp":
        return _fixed(16384, 32, 64, 1, 32, 8, 128)
    raise KeyError(name)


def custom_shape(prompt_lens: Sequence[int], branch_lens: Sequence[Sequence[int]],
                 hq: int, hkv: int, d: int) -> GroupShape:
    return GroupShape(tuple(int(p) for p in prompt_lens),
                      tuple(tuple(int(x) for x in r) for r in branch_lens), hq, hkv, d)


# ---------------------------------------------------------------------------
# fp32 -> bf16 (round to nearest even) on bit patterns.
# ---------------------------------------------------------------------------

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """RNE fp32 -> bf16, returned as uint16 bit patterns (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def bf16_bits_to_f64(b: np.ndarray) -> np.ndarray:
    return bf16_bits_to_f32(b).astype(np.float64)


CHUNK_ROWS = 2048


def _round_bf16(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bits, round to nearest even (torch's conversion; equal to
    ``f32_to_bf16_bits``, which the tests pin)."""
    import torch
    return torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def _draw_bf16(seed: int, tensor: int, shape, mult: Optional[float], pool) -> np.ndarray:
    """The packed [rows, ...] tensor `tensor` of a workload, chunk by chunk from
    independent streams, multiplied by `mult` in fp32, rounded to bf16."""
    out = np.empty(shape, dtype=np.uint16)
    rows = shape[0]
    per_row = int(np.prod(shape[1:]))
    m = None if mult is None else np.float32(mult)

    def chunk(c):
        r0 = c * CHUNK_ROWS
        n = min(CHUNK_ROWS, rows - r0)
        g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, tensor, c])))
        x = g.standard_normal(n * per_row, dtype=np.float32)
        if m is not None:
            x *= m
        out[r0:r0 + n] = _round_bf16(x).reshape((n,) + tuple(shape[1:]))

    list(pool.map(chunk, range((rows + CHUNK_ROWS - 1) // CHUNK_ROWS)))
    return out


@dataclasses.dataclass
class GroupInputs:
    shape: GroupShape
    q_p: np.ndarray
    k_p: np.ndarray
    v_p: np.ndarray
    q_r: np.ndarray
    k_r: np.ndarray
    v_r: np.ndarray
    do_p: np.ndarray
    do_r: np.ndarray


def make_inputs(shape: GroupShape, seed: int, qk_mult: Optional[float] = None, threads: Optional[int] = None) -> GroupInputs:
    """Draw the eight packed bf16 tensors. ``qk_mult`` overrides the 1/sqrt(d)
    multiplier of Q and K (V keeps 1/sqrt(d)); ``qk_mult=1.0`` gives the "sharp"
    inputs with logit std about 1."""
    import concurrent.futures as cf
    import os
    hq, hkv, d = shape.num_q_heads, shape.num_kv_heads, shape.head_dim
    tp, tr = shape.total_prompt, shape.total_resp
    inv = 1.0 / math.sqrt(d)
    mq = inv if qk_mult is None else qk_mult
    specs = [((tp, hq, d), mq), ((tp, hkv, d), mq), ((tp, hkv, d), inv),
             ((tr, hq, d), mq), ((tr, hkv, d), mq), ((tr, hkv, d), inv),
             ((tp, hq, d), None), ((tr, hq, d), None)]
    import torch
    n = threads or min(16, len(os.sched_getaffinity(0)))
    prev = torch.get_num_threads()
    torch.set_num_threads(1)  # parallelism comes from the chunk threads
    try:
        with cf.ThreadPoolExecutor(max_workers=n) as pool:
            arrs = [_draw_bf16(seed, t, sh, mult, pool) for t, (sh, mult) in enumerate(specs)]
    finally:
        torch.set_num_threads(prev)
    return GroupInputs(shape, *arrs)


def make_config(name: str) -> GroupInputs:
    """Shape and tensors of a named workload."""
    return make_inputs(config_shape(name), CONFIG_SEEDS[name])


def random_shape(rng: np.random.Generator, max_groups: int = 3, max_p: int = 300, max_g: int = 4,
                 max_r: int = 200, heads=((4, 4, 64), (8, 2, 128))) -> GroupShape:
    """A small ragged shape for property tests (lengths >= 1)."""
    ng = int(rng.integers(1, max_groups + 1))
    hq, hkv, d = heads[int(rng.integers(0, len(heads)))]
    ps = [int(rng.integers(1, max_p + 1)) for _ in range(ng)]
    rs = [tuple(int(rng.integers(1, max_r + 1)) for _ in range(int(rng.integers(1, max_g + 1))))
          for _ in range(ng)]
    return custom_shape(ps, rs, hq, hkv, d)
