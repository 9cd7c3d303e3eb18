"""Plain fp64 definitions of shared-prompt group attention (test infrastructure).

Notation follows the paper: a replay tree T = (P, {R_i}) has one prompt P and G
response branches R_i (§2.1, §3.1). For one head, attention is
O = softmax(Q K^T / sqrt(D_h) + M) V (§2.2). A token of branch i sees the whole
prompt and its own prefix, never a sibling branch (§2.2; Eq. 1,
KV(R_{i,t}) = KV_P ∪ KV(R_{i,<t})). Positions here are input positions:
query row r sees keys j <= r (the standard causal mask of the flattened
sequence [P; R_i]).

Conventions (readings of the paper where it leaves a choice):
* LSE is the natural log of the sum of exp of the *scaled* logits over the
  visible keys; a row with no visible key has LSE = -inf and O = 0.
* The partial softmax state of §3.3, (m, l, O_acc), is carried as
  (O = O_acc / l, LSE = m + ln l), which holds the same information.
* GQA: KV head k serves query heads k*g .. k*g+g-1 with g = Hq / Hkv.
* Backward of L = sum(dO * O): D_r = sum_c dO_rc O_rc, dP = dO V^T,
  dS = P * (dP - D), dQ = s dS K, dK = s dS^T Q, dV = P^T dO.

All arrays are float64. Inputs are the bf16 values upcast exactly.
"""
from __future__ import annotations

import multiprocessing as mp
from typing import Dict, Optional, Sequence

import numpy as np

# rows per query block in the blocked causal loops; keeps a block's score
# matrix under about 64 MiB for sequences up to 32k keys
_ROW_BLOCK = 256


# ---------------------------------------------------------------------------
# One head, explicit mask (the definitions themselves)
# ---------------------------------------------------------------------------

def attend_fwd(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float,
               visible: np.ndarray):
    """Masked softmax attention of one head (§2.2).

    q [n,d], k [m,d], v [m,d]; visible bool [n,m], True where key j is visible
    to query r. Returns O [n,d] and LSE [n]."""
    s = np.where(visible, scale * (q @ k.T), -np.inf)
    m = np.max(s, axis=1) if s.shape[1] else np.full(s.shape[0], -np.inf)
    m0 = np.where(np.isfinite(m), m, 0.0)
    e = np.exp(s - m0[:, None])                      # masked entries give exactly 0
    l = e.sum(axis=1)
    has = l > 0
    lse = np.where(has, m0 + np.log(np.where(has, l, 1.0)), -np.inf)
    p = e / np.where(has, l, 1.0)[:, None]
    return p @ v, lse


def attend_bwd(q, k, v, o, lse, do, scale: float, visible: np.ndarray):
    """Gradients of sum(dO * O) for the attention of ``attend_fwd``.

    ``o`` and ``lse`` are the row outputs the probabilities are normalised by
    (for a merged replay row: the merged output and merged LSE)."""
    lse0 = np.where(np.isfinite(lse), lse, 0.0)
    arg = np.where(visible, scale * (q @ k.T) - lse0[:, None], -np.inf)
    p = np.exp(arg)
    dsum = np.sum(do * o, axis=1)                    # D_r
    dp = do @ v.T
    ds = p * (dp - dsum[:, None])
    return scale * (ds @ k), scale * (ds.T @ q), p.T @ do


def causal_mask(n_q: int, n_k: int, q_offset: int = 0) -> np.ndarray:
    """visible[r, j] = (j <= r + q_offset): query r sits at position r + q_offset
    of a sequence whose keys start at position 0."""
    r = np.arange(n_q)[:, None] + q_offset
    j = np.arange(n_k)[None, :]
    return j <= r


# ---------------------------------------------------------------------------
# Blocked causal attention over one sequence (same definitions, row blocks)
# ---------------------------------------------------------------------------

def causal_fwd(q, k, v, scale):
    """Causal attention over one sequence, query rows in blocks."""
    n, d = q.shape
    o = np.empty((n, v.shape[1]))
    lse = np.empty(n)
    for r0 in range(0, n, _ROW_BLOCK):
        r1 = min(n, r0 + _ROW_BLOCK)
        o[r0:r1], lse[r0:r1] = attend_fwd(q[r0:r1], k[:r1], v[:r1], scale,
                                          causal_mask(r1 - r0, r1, r0))
    return o, lse


def causal_bwd(q, k, v, o, lse, do, scale):
    n, d = q.shape
    dq = np.empty_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    for r0 in range(0, n, _ROW_BLOCK):
        r1 = min(n, r0 + _ROW_BLOCK)
        a, b, c = attend_bwd(q[r0:r1], k[:r1], v[:r1], o[r0:r1], lse[r0:r1], do[r0:r1],
                             scale, causal_mask(r1 - r0, r1, r0))
        dq[r0:r1] = a
        dk[:r1] += b
        dv[:r1] += c
    return dq, dk, dv


# ---------------------------------------------------------------------------
# The merge of partial softmax states (§3.3)
# ---------------------------------------------------------------------------

def lse_merge(o_parts: np.ndarray, lse_parts: np.ndarray):
    """Merge n partial states of the same query rows.

    o_parts [n, ..., d] are outputs normalised within each part, lse_parts
    [n, ...] their LSEs. Returns (O, LSE) with LSE = ln sum_k exp(LSE_k) and
    O = sum_k exp(LSE_k - LSE) O_k. Parts with LSE = -inf carry weight 0; if
    every part is -inf the result is O = 0, LSE = -inf."""
    lse_parts = np.asarray(lse_parts, dtype=np.float64)
    m = np.max(lse_parts, axis=0)
    m0 = np.where(np.isfinite(m), m, 0.0)
    w = np.exp(lse_parts - m0)                       # exp(-inf) = 0
    tot = w.sum(axis=0)
    has = tot > 0
    lse = np.where(has, m0 + np.log(np.where(has, tot, 1.0)), -np.inf)
    coef = w / np.where(has, tot, 1.0)
    o = np.sum(coef[..., None] * o_parts, axis=0)
    return o, lse


def prompt_grad_sum(self_part: Optional[np.ndarray], parts: Sequence[np.ndarray]):
    """Eq. 2: the prompt-KV gradient is the prefill's own contribution plus the
    sum over branches (or chunks of branches) of their contributions, summed in
    index order."""
    out = np.zeros_like(parts[0]) if self_part is None else np.array(self_part, dtype=np.float64)
    for p in parts:
        out = out + p
    return out


# ---------------------------------------------------------------------------
# Flattened reference: each branch as the causal sequence [P; R_i]
# ---------------------------------------------------------------------------

def _flat_unit(args):
    (qp, kp, vp, qr, kr, vr, dop, dor, w, scale) = args
    q = np.concatenate([qp, qr])
    k = np.concatenate([kp, kr])
    v = np.concatenate([vp, vr])
    do = np.concatenate([w * dop, dor])
    o, lse = causal_fwd(q, k, v, scale)
    dq, dk, dv = causal_bwd(q, k, v, o, lse, do, scale)
    return o, lse, dq, dk, dv


_POOL_ARGS = None


def _flat_unit_idx(i):
    return _flat_unit(_POOL_ARGS[i])


def flattened_fwd_bwd(cu_prompt, cu_branch, cu_resp, num_q_heads: int, num_kv_heads: int,
                      scale: float, q_p, k_p, v_p, q_r, k_r, v_r, do_p, do_r,
                      weights: Optional[Sequence[float]] = None, workers: int = 1,
                      check_copies: bool = True) -> Dict[str, np.ndarray]:
    """Flattened per-branch causal attention, forward and backward (§2.1).

    Packed layouts: q_p [T_P,Hq,d], k_p/v_p [T_P,Hkv,d], q_r [T_R,Hq,d],
    k_r/v_r [T_R,Hkv,d], do_p/do_r like q. Copy i of group g is the sequence
    [P_g; R_i] and receives the upstream gradient [w_i dO_P; dO_{R_i}] with
    w_i = weights[branch] (default 1/G_g). Prompt results are assembled from
    the copies: O_P, LSE_P from the first copy; dQ_P, dK_P, dV_P summed over
    copies (and dK, dV over the query heads of each KV head) in a fixed order.

    Returns float64 arrays o_p, lse_p [Hq,T_P], o_r, lse_r [Hq,T_R], dq_p, dk_p,
    dv_p, dq_r, dk_r, dv_r."""
    cu_prompt = np.asarray(cu_prompt)
    cu_branch = np.asarray(cu_branch)
    cu_resp = np.asarray(cu_resp)
    hq, hkv = num_q_heads, num_kv_heads
    gq = hq // hkv
    tp, tr = q_p.shape[0], q_r.shape[0]
    d = q_p.shape[2]
    units, keys = [], []
    for g in range(len(cu_prompt) - 1):
        p0, p1 = int(cu_prompt[g]), int(cu_prompt[g + 1])
        b0, b1 = int(cu_branch[g]), int(cu_branch[g + 1])
        for h in range(hq):
            kh = h // gq
            for b in range(b0, b1):
                r0, r1 = int(cu_resp[b]), int(cu_resp[b + 1])
                w = (1.0 / (b1 - b0)) if weights is None else float(weights[b])
                units.append((q_p[p0:p1, h], k_p[p0:p1, kh], v_p[p0:p1, kh],
                              q_r[r0:r1, h], k_r[r0:r1, kh], v_r[r0:r1, kh],
                              do_p[p0:p1, h], do_r[r0:r1, h], w, scale))
                keys.append((g, h, b))
    if workers > 1 and len(units) > 1:
        global _POOL_ARGS
        _POOL_ARGS = units
        order = sorted(range(len(units)), key=lambda i: -(units[i][0].shape[0] + units[i][3].shape[0]))
        with mp.get_context("fork").Pool(workers) as pool:
            got = dict(zip(order, pool.map(_flat_unit_idx, order, chunksize=1)))
        results = [got[i] for i in range(len(units))]
        _POOL_ARGS = None
    else:
        results = [_flat_unit(u) for u in units]

    out = {
        "o_p": np.zeros((tp, hq, d)), "lse_p": np.zeros((hq, tp)),
        "o_r": np.zeros((tr, hq, d)), "lse_r": np.zeros((hq, tr)),
        "dq_p": np.zeros((tp, hq, d)), "dk_p": np.zeros((tp, hkv, d)), "dv_p": np.zeros((tp, hkv, d)),
        "dq_r": np.zeros((tr, hq, d)), "dk_r": np.zeros((tr, hkv, d)), "dv_r": np.zeros((tr, hkv, d)),
    }
    seen_prompt = set()
    # fixed summation order: units are visited in (group, head, branch) order
    for (g, h, b), (o, lse, dq, dk, dv) in zip(keys, results):
        p0, p1 = int(cu_prompt[g]), int(cu_prompt[g + 1])
        r0, r1 = int(cu_resp[b]), int(cu_resp[b + 1])
        P = p1 - p0
        kh = h // gq
        if (g, h) not in seen_prompt:
            seen_prompt.add((g, h))
            out["o_p"][p0:p1, h] = o[:P]
            out["lse_p"][h, p0:p1] = lse[:P]
        elif check_copies:
            ref = out["o_p"][p0:p1, h]
            err = np.linalg.norm(o[:P] - ref) / max(np.linalg.norm(ref), 1e-300)
            if err > 1e-13:
                raise AssertionError(f"flattened copies disagree on prompt rows: {err}")
        out["o_r"][r0:r1, h] = o[P:]
        out["lse_r"][h, r0:r1] = lse[P:]
        out["dq_p"][p0:p1, h] += dq[:P]
        out["dq_r"][r0:r1, h] = dq[P:]
        out["dk_p"][p0:p1, kh] += dk[:P]
        out["dv_p"][p0:p1, kh] += dv[:P]
        out["dk_r"][r0:r1, kh] += dk[P:]
        out["dv_r"][r0:r1, kh] += dv[P:]
    return out


# ---------------------------------------------------------------------------
# Shared-prompt decomposition (§3.2-§3.3, Eq. 1-2); used to check exactness
# ---------------------------------------------------------------------------

def shared_fwd_bwd(cu_prompt, cu_branch, cu_resp, num_q_heads: int, num_kv_heads: int,
                   scale: float, q_p, k_p, v_p, q_r, k_r, v_r, do_p, do_r) -> Dict[str, np.ndarray]:
    """The method's decomposition in fp64.

    Forward: prompt prefill once (causal over P); each branch as a prompt
    partial (all P keys visible) and a branch-local causal partial, merged with
    ``lse_merge``. Backward: both partials are differentiated with the merged O
    and LSE; the branch's prompt-key gradients are the seeds; the prompt
    gradient is the prefill contribution plus the seeds of every branch (Eq. 2).

    Returns the same keys as ``flattened_fwd_bwd`` plus ``dk_p_self``,
    ``dv_p_self`` and ``seed_k``/``seed_v`` [num_branches, P_g-rows packed like
    k_p] (each branch's prompt-key gradient, summed over the query heads of a KV
    head)."""
    cu_prompt = np.asarray(cu_prompt)
    cu_branch = np.asarray(cu_branch)
    cu_resp = np.asarray(cu_resp)
    hq, hkv = num_q_heads, num_kv_heads
    gq = hq // hkv
    tp, tr = q_p.shape[0], q_r.shape[0]
    d = q_p.shape[2]
    nb = len(cu_resp) - 1
    out = {
        "o_p": np.zeros((tp, hq, d)), "lse_p": np.zeros((hq, tp)),
        "o_r": np.zeros((tr, hq, d)), "lse_r": np.zeros((hq, tr)),
        "dq_p": np.zeros((tp, hq, d)), "dq_r": np.zeros((tr, hq, d)),
        "dk_r": np.zeros((tr, hkv, d)), "dv_r": np.zeros((tr, hkv, d)),
        "dk_p_self": np.zeros((tp, hkv, d)), "dv_p_self": np.zeros((tp, hkv, d)),
        "seed_k": np.zeros((nb, tp, hkv, d)), "seed_v": np.zeros((nb, tp, hkv, d)),
    }
    for g in range(len(cu_prompt) - 1):
        p0, p1 = int(cu_prompt[g]), int(cu_prompt[g + 1])
        for h in range(hq):
            kh = h // gq
            Kp, Vp = k_p[p0:p1, kh], v_p[p0:p1, kh]
            # prefill, once per group and head
            o, lse = causal_fwd(q_p[p0:p1, h], Kp, Vp, scale)
            out["o_p"][p0:p1, h] = o
            out["lse_p"][h, p0:p1] = lse
            dq, dk, dv = causal_bwd(q_p[p0:p1, h], Kp, Vp, o, lse, do_p[p0:p1, h], scale)
            out["dq_p"][p0:p1, h] = dq
            out["dk_p_self"][p0:p1, kh] += dk
            out["dv_p_self"][p0:p1, kh] += dv
            for b in range(int(cu_branch[g]), int(cu_branch[g + 1])):
                r0, r1 = int(cu_resp[b]), int(cu_resp[b + 1])
                Q, Kr, Vr, dO = q_r[r0:r1, h], k_r[r0:r1, kh], v_r[r0:r1, kh], do_r[r0:r1, h]
                R, P = r1 - r0, p1 - p0
                vis_a = np.ones((R, P), dtype=bool)
                vis_b = causal_mask(R, R)
                oa, la = attend_fwd(Q, Kp, Vp, scale, vis_a)
                ob, lb = attend_fwd(Q, Kr, Vr, scale, vis_b)
                o_m, l_m = lse_merge(np.stack([oa, ob]), np.stack([la, lb]))
                out["o_r"][r0:r1, h] = o_m
                out["lse_r"][h, r0:r1] = l_m
                dqa, dka, dva = attend_bwd(Q, Kp, Vp, o_m, l_m, dO, scale, vis_a)
                dqb, dkb, dvb = attend_bwd(Q, Kr, Vr, o_m, l_m, dO, scale, vis_b)
                out["dq_r"][r0:r1, h] = dqa + dqb
                out["dk_r"][r0:r1, kh] += dkb
                out["dv_r"][r0:r1, kh] += dvb
                out["seed_k"][b, p0:p1, kh] += dka
                out["seed_v"][b, p0:p1, kh] += dva
    # Eq. 2: prefill contribution first, then the branches in index order
    out["dk_p"] = prompt_grad_sum(out["dk_p_self"], list(out["seed_k"]))
    out["dv_p"] = prompt_grad_sum(out["dv_p_self"], list(out["seed_v"]))
    return out
