"""Single-row references for full-size workloads (test infrastructure).

The full flattened oracle costs about 14*d*Hq*(valid pairs) fp64 flops, which is
out of reach for the large workloads. The definitions of ``attention`` are
applied here to chosen query rows (output, LSE, dQ of those rows) or chosen key
rows (dK, dV of those keys, which needs the LSE and D of every query that sees
them). The visible key set of a row follows Eq. 1: a prompt row at position p
sees prompt keys 0..p; a response row at position t of branch i sees all
prompt keys and keys 0..t of branch i.

Inputs are the packed bf16 bit patterns (uint16); only the rows a computation
needs are decoded to float64.
"""
from __future__ import annotations

from typing import Dict, Sequence

import numpy as np

_BLOCK = 256


def _block_rows(n_keys: int) -> int:
    """Query rows per block against ``n_keys`` keys: at most 2^21 scores (16 MB
    of float64 per temporary), so the temporaries of one block are reused from
    the heap instead of being mapped and faulted in afresh for every block."""
    return int(max(16, min(_BLOCK, (1 << 21) // max(n_keys, 1))))


def _f64(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> float64 (exact)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def _group_of_prompt_row(cu_prompt, row):
    return int(np.searchsorted(cu_prompt, row, side="right") - 1)


def _branch_of_resp_row(cu_resp, row):
    return int(np.searchsorted(cu_resp, row, side="right") - 1)


def _group_of_branch(cu_branch, b):
    return int(np.searchsorted(cu_branch, b, side="right") - 1)


def _rows_block(q, do, k, v, visible, scale):
    """LSE, O, P and dS of a block of query rows against a key set (definitions
    of §2.2; D from this block's own exact O)."""
    s = np.where(visible, scale * (q @ k.T), -np.inf)
    m = s.max(axis=1)
    e = np.exp(s - m[:, None])
    l = e.sum(axis=1)
    lse = m + np.log(l)
    p = e / l[:, None]
    o = p @ v
    dsum = np.sum(do * o, axis=1)
    ds = p * (do @ v.T - dsum[:, None])
    return lse, o, p, ds


def _keyset_prompt(t, g, kh, upto):
    p0 = int(t.cu_prompt[g])
    return _f64(t.k_p[p0:p0 + upto, kh]), _f64(t.v_p[p0:p0 + upto, kh])


def query_rows(t, kind: str, rows: Sequence[int], head: int) -> Dict[str, np.ndarray]:
    """O, LSE and dQ of packed query rows ``rows`` of query head ``head``.

    ``t`` carries cu_prompt, cu_branch, cu_resp (int arrays), num_q_heads,
    num_kv_heads, head_dim and the eight packed bf16 arrays (q_p .. do_r).
    ``kind`` is "prompt" or "resp". Returns float64 o [n,d], lse [n], dq [n,d]."""
    scale = 1.0 / np.sqrt(t.head_dim)
    kh = head // (t.num_q_heads // t.num_kv_heads)
    n = len(rows)
    o = np.zeros((n, t.head_dim))
    lse = np.zeros(n)
    dq = np.zeros((n, t.head_dim))
    for i, r in enumerate(rows):
        r = int(r)
        if kind == "prompt":
            g = _group_of_prompt_row(t.cu_prompt, r)
            pos = r - int(t.cu_prompt[g])
            k, v = _keyset_prompt(t, g, kh, pos + 1)
            q, do = _f64(t.q_p[r:r + 1, head]), _f64(t.do_p[r:r + 1, head])
        else:
            b = _branch_of_resp_row(t.cu_resp, r)
            g = _group_of_branch(t.cu_branch, b)
            pos = r - int(t.cu_resp[b])
            P = int(t.cu_prompt[g + 1] - t.cu_prompt[g])
            kp, vp = _keyset_prompt(t, g, kh, P)
            r0 = int(t.cu_resp[b])
            k = np.concatenate([kp, _f64(t.k_r[r0:r0 + pos + 1, kh])])
            v = np.concatenate([vp, _f64(t.v_r[r0:r0 + pos + 1, kh])])
            q, do = _f64(t.q_r[r:r + 1, head]), _f64(t.do_r[r:r + 1, head])
        vis = np.ones((1, k.shape[0]), dtype=bool)
        l, oo, _, ds = _rows_block(q, do, k, v, vis, scale)
        o[i], lse[i] = oo[0], l[0]
        dq[i] = scale * (ds @ k)[0]
    return {"o": o, "lse": lse, "dq": dq}


def _key_unit(t, kind, cols, kv_head, h, seg):
    """dK, dV of the key columns ``cols`` (positions inside the key set of
    ``seg``) from the queries of one query head ``h`` in one range of query
    rows: seg = ("prefill", g, a0, a1) the prompt rows a0 .. a1-1 of group g
    (keys = that prompt, causal), ("branch", b, a0, a1) the rows a0 .. a1-1 of
    branch b (keys = its group's prompt followed by its own prefix). For kind
    "resp" the columns are positions inside branch b's own keys."""
    scale = 1.0 / np.sqrt(t.head_dim)
    d = t.head_dim
    cols = np.asarray(cols)
    dk = np.zeros((len(cols), d))
    dv = np.zeros((len(cols), d))
    a0, a1 = seg[2], seg[3]
    if seg[0] == "prefill":
        g = seg[1]
        p0, p1 = int(t.cu_prompt[g]), int(t.cu_prompt[g + 1])
        P = p1 - p0
        kp, vp = _keyset_prompt(t, g, kv_head, P)
        step = _block_rows(P)
        for a in range(a0, a1, step):
            bnd = min(a1, a + step)
            q = _f64(t.q_p[p0 + a:p0 + bnd, h])
            do = _f64(t.do_p[p0 + a:p0 + bnd, h])
            vis = np.arange(bnd)[None, :] <= np.arange(a, bnd)[:, None]
            _, _, p, ds = _rows_block(q, do, kp[:bnd], vp[:bnd], vis, scale)
            sel = cols < bnd
            dk[sel] += scale * (ds[:, cols[sel]].T @ q)
            dv[sel] += p[:, cols[sel]].T @ do
        return dk, dv
    b = seg[1]
    g = _group_of_branch(t.cu_branch, b)
    r0, r1 = int(t.cu_resp[b]), int(t.cu_resp[b + 1])
    P = int(t.cu_prompt[g + 1] - t.cu_prompt[g])
    kp, vp = _keyset_prompt(t, g, kv_head, P)
    kr, vr = _f64(t.k_r[r0:r1, kv_head]), _f64(t.v_r[r0:r1, kv_head])
    kk, vv = np.concatenate([kp, kr]), np.concatenate([vp, vr])
    c = cols if kind == "prompt" else cols + P
    step = _block_rows(P + r1 - r0)
    for a in range(a0, a1, step):
        bnd = min(a1, a + step)
        q = _f64(t.q_r[r0 + a:r0 + bnd, h])
        do = _f64(t.do_r[r0 + a:r0 + bnd, h])
        vis = np.concatenate([np.ones((bnd - a, P), dtype=bool),
                              np.arange(r1 - r0)[None, :] <= np.arange(a, bnd)[:, None]], axis=1)
        _, _, p, ds = _rows_block(q, do, kk, vv, vis, scale)
        sel = np.ones(len(cols), dtype=bool) if kind == "prompt" else cols < bnd
        dk[sel] += scale * (ds[:, c[sel]].T @ q)
        dv[sel] += p[:, c[sel]].T @ do
    return dk, dv


# query rows per term of key_rows (terms are computed independently and
# added in order)
_TERM_ROWS = 2048


def _ranges(a0, a1):
    return [(a, min(a1, a + _TERM_ROWS)) for a in range(a0, a1, _TERM_ROWS)]


_UNIT_ARGS = None


def _key_unit_idx(i):
    # one BLAS thread per worker process: the pool supplies the parallelism
    from threadpoolctl import threadpool_limits
    with threadpool_limits(1):
        return _key_unit(*_UNIT_ARGS[i])


def key_rows(t, kind: str, rows: Sequence[int], kv_head: int, workers: int = 1) -> Dict[str, np.ndarray]:
    """dK and dV of packed key rows ``rows`` of KV head ``kv_head``, summed over
    the query heads of that KV head and over every query that sees the key.

    kind "prompt": all rows must belong to one group; the queries are the
    group's prompt rows at or after the earliest sampled key, plus every
    response row of the group (this is the total of Eq. 2: the prefill
    contribution plus every branch's contribution). kind "resp": all rows must
    belong to one branch; the queries are that branch's rows at or after the
    earliest sampled key.

    The sum runs over (query head, range of query rows) terms in a fixed
    order: for each query head, the prompt rows first, then the branches in
    index order (Eq. 2's order), each in ranges of _TERM_ROWS rows. ``workers``
    > 1 computes the terms in a process pool and adds them in the same order,
    so the result is the same bit for bit."""
    gq = t.num_q_heads // t.num_kv_heads
    rows = [int(r) for r in rows]
    d = t.head_dim
    units = []
    if kind == "prompt":
        g = _group_of_prompt_row(t.cu_prompt, rows[0])
        p0, p1 = int(t.cu_prompt[g]), int(t.cu_prompt[g + 1])
        assert all(p0 <= r < p1 for r in rows)
        cols = np.array([r - p0 for r in rows])
        for h in range(kv_head * gq, kv_head * gq + gq):
            for a, z in _ranges(int(cols.min()), p1 - p0):
                units.append((t, kind, cols, kv_head, h, ("prefill", g, a, z)))
            for b in range(int(t.cu_branch[g]), int(t.cu_branch[g + 1])):
                for a, z in _ranges(0, int(t.cu_resp[b + 1] - t.cu_resp[b])):
                    units.append((t, kind, cols, kv_head, h, ("branch", b, a, z)))
    else:
        b = _branch_of_resp_row(t.cu_resp, rows[0])
        r0, r1 = int(t.cu_resp[b]), int(t.cu_resp[b + 1])
        assert all(r0 <= r < r1 for r in rows)
        cols = np.array([r - r0 for r in rows])
        for h in range(kv_head * gq, kv_head * gq + gq):
            for a, z in _ranges(int(cols.min()), r1 - r0):
                units.append((t, kind, cols, kv_head, h, ("branch", b, a, z)))
    if workers > 1 and len(units) > 1:
        import multiprocessing as mp
        global _UNIT_ARGS
        _UNIT_ARGS = units
        try:
            with mp.get_context("fork").Pool(min(workers, len(units))) as pool:
                parts = pool.map(_key_unit_idx, range(len(units)), chunksize=1)
        finally:
            _UNIT_ARGS = None
    else:
        parts = [_key_unit(*u) for u in units]
    dk = np.zeros((len(rows), d))
    dv = np.zeros((len(rows), d))
    for a, b in parts:
        dk = dk + a
        dv = dv + b
    return {"dk": dk, "dv": dv}
