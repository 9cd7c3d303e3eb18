"""Pins of the fp64 oracle against things other than itself (CPU only).

* closed forms: the log-sum-exp merge against one softmax over the joined keys
  (§3.3), and the Q = 0 probe whose LSE is ln(#visible keys) and whose output
  is the mean of the visible values (pins the Eq. 1 mask: diagonal, prompt
  column, no sibling keys);
* a library routine: torch's scaled_dot_product_attention and autograd on CPU
  in float64 for G = 1 (a single flattened causal sequence) with GQA via
  repeat_interleave;
* brute force: pure-Python loops over a tiny sequence;
* finite differences of L = sum(dO * O) for every gradient;
* invariants of the method: the shared decomposition equals the flattened
  reference (§3.2, §3.3) and the prompt gradient is the prefill part plus the
  sum of per-branch parts (Eq. 2); the split of dO_P over copies does not
  change totals; the per-branch seeds equal a flattened copy with no prompt-row
  gradient.
"""
import math

import numpy as np
import pytest

from oracle import attention as A
from oracle import sampled as S
from paper_2609_33133_amd import inputs as I


def f64_inputs(gi):
    c = I.bf16_bits_to_f64
    return [c(x) for x in (gi.q_p, gi.k_p, gi.v_p, gi.q_r, gi.k_r, gi.v_r, gi.do_p, gi.do_r)]


def run(fn, gi, **kw):
    s = gi.shape
    return fn(s.cu_prompt, s.cu_branch, s.cu_resp, s.num_q_heads, s.num_kv_heads, s.scale,
              *f64_inputs(gi), **kw)


def rel(a, b):
    nb = np.linalg.norm(b)
    return np.linalg.norm(a - b) / (nb if nb > 0 else 1.0)


TINY = I.custom_shape([7], [[5, 1, 4]], 4, 2, 8)        # P=7, G=3, R=(5,1,4), Hq=4, Hkv=2, d=8
SMALL = I.custom_shape([13, 6], [[9, 3], [4, 11, 2]], 4, 2, 16)


# --------------------------------------------------------------------------- inputs

def test_bf16_rne_matches_torch():
    import torch
    rng = np.random.default_rng(1)
    x = np.concatenate([rng.standard_normal(10000).astype(np.float32) * 3,
                        np.array([1.00390625, 1.01171875, -1.00390625, 0.0, -0.0, 65504.0], np.float32)])
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(I.f32_to_bf16_bits(x), ref)
    assert np.array_equal(I.bf16_bits_to_f32(ref), torch.from_numpy(ref.view(np.int16)).view(torch.bfloat16).float().numpy())


def test_ragged_sampler_reading():
    rng = np.random.Generator(np.random.PCG64(7))
    ps, rs, attempt = I.ragged_lengths(rng)
    assert attempt == 9
    assert ps[0] == 11759 and rs[0] == (427, 615, 1146, 1004)
    s = I.config_shape("ragged")
    assert s.num_groups == 16 and s.num_branches == 148
    assert s.total_prompt == 199648 and s.total_resp == 828181
    assert s.total_prompt + s.total_resp <= I.TOKEN_CAP


def test_valid_pair_counts_brute_force():
    s = SMALL
    vp = s.valid_pairs()
    # count visible pairs by building every mask explicitly
    pre = sum(int(A.causal_mask(p, p).sum()) for p in s.prompt_lens)
    flat = sum(int(A.causal_mask(p + r, p + r).sum()) for p, rs in zip(s.prompt_lens, s.branch_lens) for r in rs)
    assert vp["prefill"] == pre and vp["flattened"] == flat
    assert vp["flattened"] - vp["shared"] == sum((len(rs) - 1) * p * (p + 1) // 2
                                                 for p, rs in zip(s.prompt_lens, s.branch_lens))


# --------------------------------------------------------------------------- merge

def test_merge_equals_softmax_over_joined_keys():
    rng = np.random.default_rng(2)
    n, d = 9, 16
    q = rng.standard_normal((n, d))
    ka, va = rng.standard_normal((5, d)), rng.standard_normal((5, d))
    kb, vb = rng.standard_normal((11, d)), rng.standard_normal((11, d))
    s = 0.7
    oa, la = A.attend_fwd(q, ka, va, s, np.ones((n, 5), bool))
    ob, lb = A.attend_fwd(q, kb, vb, s, np.ones((n, 11), bool))
    om, lm = A.lse_merge(np.stack([oa, ob]), np.stack([la, lb]))
    # the same rows as one softmax, written out with math.exp
    for r in range(n):
        logits = [s * float(q[r] @ k) for k in np.concatenate([ka, kb])]
        z = sum(math.exp(x) for x in logits)
        vals = np.concatenate([va, vb])
        o = sum(math.exp(x) / z * vals[j] for j, x in enumerate(logits))
        assert abs(lm[r] - math.log(z)) < 1e-13
        assert np.max(np.abs(om[r] - o)) < 1e-13


def test_merge_commutative_associative_identity():
    rng = np.random.default_rng(3)
    o = rng.standard_normal((3, 6, 4))
    l = rng.standard_normal((3, 6)) * 5
    o01, l01 = A.lse_merge(o[[0, 1]], l[[0, 1]])
    o10, l10 = A.lse_merge(o[[1, 0]], l[[1, 0]])
    assert np.max(np.abs(o01 - o10)) < 1e-13 and np.max(np.abs(l01 - l10)) < 1e-13
    left_o, left_l = A.lse_merge(np.stack([o01, o[2]]), np.stack([l01, l[2]]))
    o12, l12 = A.lse_merge(o[[1, 2]], l[[1, 2]])
    right_o, right_l = A.lse_merge(np.stack([o[0], o12]), np.stack([l[0], l12]))
    all_o, all_l = A.lse_merge(o, l)
    for a, b in ((left_o, right_o), (left_o, all_o), (left_l, right_l), (left_l, all_l)):
        assert np.max(np.abs(a - b)) < 1e-13
    # a part with LSE = -inf is the identity, exactly
    io, il = A.lse_merge(np.stack([o[0], rng.standard_normal((6, 4))]),
                         np.stack([l[0], np.full(6, -np.inf)]))
    assert np.array_equal(io, o[0]) and np.array_equal(il, l[0])
    # every part empty: O = 0, LSE = -inf, never NaN
    zo, zl = A.lse_merge(o[:2], np.full((2, 6), -np.inf))
    assert np.all(zo == 0) and np.all(zl == -np.inf)


def test_prompt_grad_sum_order_and_values():
    rng = np.random.default_rng(4)
    parts = [rng.standard_normal((3, 2)) for _ in range(4)]
    base = rng.standard_normal((3, 2))
    got = A.prompt_grad_sum(base, parts)
    exp = base.copy()
    for r in range(3):
        for c in range(2):
            acc = base[r, c]
            for p in parts:
                acc = acc + p[r, c]
            exp[r, c] = acc
    assert np.array_equal(got, exp)            # same order => bit-identical
    assert np.array_equal(A.prompt_grad_sum(None, parts), sum(parts[1:], parts[0]))


# --------------------------------------------------------------------------- brute force

def test_attend_brute_force_tiny():
    rng = np.random.default_rng(5)
    n, d = 6, 3
    q, k, v = (rng.standard_normal((n, d)) for _ in range(3))
    s = 0.5
    o, lse = A.causal_fwd(q, k, v, s)
    for r in range(n):
        logits = [s * sum(q[r][c] * k[j][c] for c in range(d)) for j in range(r + 1)]
        z = sum(math.exp(x) for x in logits)
        assert abs(lse[r] - math.log(z)) < 1e-14
        for c in range(d):
            val = sum(math.exp(logits[j]) / z * v[j][c] for j in range(r + 1))
            assert abs(o[r][c] - val) < 1e-14


def test_fully_masked_row_is_zero():
    q = np.ones((2, 4))
    o, l = A.attend_fwd(q, np.ones((3, 4)), np.ones((3, 4)), 1.0, np.zeros((2, 3), bool))
    assert np.all(o == 0) and np.all(l == -np.inf)


# --------------------------------------------------------------------------- library routine

@pytest.mark.parametrize("hq,hkv", [(4, 4), (4, 2), (6, 2)])
def test_flattened_matches_torch_sdpa_g1(hq, hkv):
    import torch
    shape = I.custom_shape([10], [[7]], hq, hkv, 8)
    gi = I.make_inputs(shape, seed=11, qk_mult=1.0)
    out = run(A.flattened_fwd_bwd, gi)
    qp, kp, vp, qr, kr, vr, dop, dor = f64_inputs(gi)
    g = hq // hkv
    q = torch.tensor(np.concatenate([qp, qr]).transpose(1, 0, 2), requires_grad=True)
    k = torch.tensor(np.concatenate([kp, kr]).transpose(1, 0, 2), requires_grad=True)
    v = torch.tensor(np.concatenate([vp, vr]).transpose(1, 0, 2), requires_grad=True)
    o = torch.nn.functional.scaled_dot_product_attention(
        q[None], k.repeat_interleave(g, 0)[None], v.repeat_interleave(g, 0)[None],
        is_causal=True, scale=shape.scale)[0]
    do = torch.tensor(np.concatenate([dop, dor]).transpose(1, 0, 2))
    (o * do).sum().backward()
    P = 10
    ot = o.detach().numpy().transpose(1, 0, 2)
    assert rel(out["o_p"], ot[:P]) < 1e-12 and rel(out["o_r"], ot[P:]) < 1e-12
    for name, t in (("dq", q), ("dk", k), ("dv", v)):
        gt = t.grad.numpy().transpose(1, 0, 2)
        assert rel(out[name + "_p"], gt[:P]) < 1e-12, name
        assert rel(out[name + "_r"], gt[P:]) < 1e-12, name
    # LSE against torch.logsumexp of the masked scaled logits
    ql = torch.tensor(np.concatenate([qp, qr]).transpose(1, 0, 2))
    kl = torch.tensor(np.concatenate([kp, kr]).transpose(1, 0, 2)).repeat_interleave(g, 0)
    logits = shape.scale * ql @ kl.transpose(1, 2)
    logits = logits.masked_fill(torch.ones(17, 17, dtype=torch.bool).triu(1), float("-inf"))
    lse = torch.logsumexp(logits, -1).numpy()
    assert np.max(np.abs(out["lse_p"] - lse[:, :P])) < 1e-12
    assert np.max(np.abs(out["lse_r"] - lse[:, P:])) < 1e-12


# --------------------------------------------------------------------------- finite differences

def test_finite_differences_tiny():
    gi = I.make_inputs(TINY, seed=12, qk_mult=1.0)
    base = f64_inputs(gi)
    s = TINY
    out = A.flattened_fwd_bwd(s.cu_prompt, s.cu_branch, s.cu_resp, 4, 2, s.scale, *base)
    dop, dor = base[6], base[7]

    def loss(arrs):
        o = A.flattened_fwd_bwd(s.cu_prompt, s.cu_branch, s.cu_resp, 4, 2, s.scale, *arrs, dop, dor,
                                check_copies=False)
        return float(np.sum(o["o_p"] * dop) + np.sum(o["o_r"] * dor))

    h = 1e-6
    rng = np.random.default_rng(13)
    names = ["dq_p", "dk_p", "dv_p", "dq_r", "dk_r", "dv_r"]
    for ti, name in enumerate(names):
        arr = base[ti]
        flat_idx = rng.choice(arr.size, size=min(50, arr.size), replace=False)
        num = np.empty(len(flat_idx))
        for n, fi in enumerate(flat_idx):
            idx = np.unravel_index(fi, arr.shape)
            plus = [x.copy() for x in base[:6]]
            minus = [x.copy() for x in base[:6]]
            plus[ti][idx] += h
            minus[ti][idx] -= h
            num[n] = (loss(plus) - loss(minus)) / (2 * h)
        ana = out[name].reshape(-1)[flat_idx]
        assert rel(ana, num) < 1e-6, (name, rel(ana, num))


# --------------------------------------------------------------------------- invariants

@pytest.mark.parametrize("shape", [TINY, SMALL])
def test_shared_equals_flattened(shape):
    gi = I.make_inputs(shape, seed=14, qk_mult=1.0)
    fl = run(A.flattened_fwd_bwd, gi)
    sh = run(A.shared_fwd_bwd, gi)
    for k in ("o_p", "o_r", "dq_p", "dq_r", "dk_p", "dv_p", "dk_r", "dv_r"):
        assert rel(sh[k], fl[k]) < 1e-12, k
    for k in ("lse_p", "lse_r"):
        assert np.max(np.abs(sh[k] - fl[k])) < 1e-12, k


def test_eq2_seeds_are_flattened_copies_without_prompt_gradient():
    """Per-branch seed i equals the prompt-key gradient of flattened copy i whose
    prompt rows get no upstream gradient (w_i = 0); the prefill contribution is
    a copy whose response rows get none."""
    s = SMALL
    gi = I.make_inputs(s, seed=15, qk_mult=1.0)
    sh = run(A.shared_fwd_bwd, gi)
    qp, kp, vp, qr, kr, vr, dop, dor = f64_inputs(gi)
    zero_w = [0.0] * s.num_branches
    fl0 = A.flattened_fwd_bwd(s.cu_prompt, s.cu_branch, s.cu_resp, 4, 2, s.scale,
                              qp, kp, vp, qr, kr, vr, dop, dor, weights=zero_w)
    assert rel(sh["seed_k"].sum(0), fl0["dk_p"]) < 1e-12
    assert rel(sh["seed_v"].sum(0), fl0["dv_p"]) < 1e-12
    # branch by branch: a shape with that branch alone
    for b in range(s.num_branches):
        g = int(np.searchsorted(s.cu_branch, b, side="right") - 1)
        p0, p1 = int(s.cu_prompt[g]), int(s.cu_prompt[g + 1])
        r0, r1 = int(s.cu_resp[b]), int(s.cu_resp[b + 1])
        one = A.flattened_fwd_bwd([0, p1 - p0], [0, 1], [0, r1 - r0], 4, 2, s.scale,
                                  qp[p0:p1], kp[p0:p1], vp[p0:p1], qr[r0:r1], kr[r0:r1], vr[r0:r1],
                                  dop[p0:p1], dor[r0:r1], weights=[0.0])
        assert rel(sh["seed_k"][b, p0:p1], one["dk_p"]) < 1e-12
        assert rel(sh["seed_v"][b, p0:p1], one["dv_p"]) < 1e-12
    # the prefill part: response rows without upstream gradient
    fl_self = A.flattened_fwd_bwd(s.cu_prompt, s.cu_branch, s.cu_resp, 4, 2, s.scale,
                                  qp, kp, vp, qr, kr, vr, dop, np.zeros_like(dor))
    assert rel(sh["dk_p_self"], fl_self["dk_p"]) < 1e-12
    assert rel(sh["dv_p_self"], fl_self["dv_p"]) < 1e-12


def test_prompt_dO_split_does_not_change_totals():
    s = SMALL
    gi = I.make_inputs(s, seed=16, qk_mult=1.0)
    even = run(A.flattened_fwd_bwd, gi)
    first = [1.0 if b in (0, 2) else 0.0 for b in range(s.num_branches)]   # e_0 per group
    one = run(A.flattened_fwd_bwd, gi, weights=first)
    for k in ("dq_p", "dk_p", "dv_p", "dq_r", "dk_r", "dv_r"):
        assert rel(one[k], even[k]) < 1e-12, k


def test_q_zero_probe_pins_the_mask():
    """Q = 0: every visible key has logit 0, so LSE = ln(#visible) and O is the
    mean of the visible values. With V[..., 0] = position label (prompt key j ->
    j, response key j -> P + j), a prompt row at p averages to p/2 and a
    response row at t averages to (P + t)/2; a sibling key or a shifted diagonal
    would change both."""
    s = SMALL
    gi = I.make_inputs(s, seed=17)
    qp, kp, vp, qr, kr, vr, dop, dor = f64_inputs(gi)
    qp[:] = 0
    qr[:] = 0
    for g in range(s.num_groups):
        p0, p1 = s.cu_prompt[g], s.cu_prompt[g + 1]
        vp[p0:p1, :, 0] = np.arange(p1 - p0)[:, None]
        for b in range(s.cu_branch[g], s.cu_branch[g + 1]):
            r0, r1 = s.cu_resp[b], s.cu_resp[b + 1]
            vr[r0:r1, :, 0] = (p1 - p0 + np.arange(r1 - r0))[:, None]
    out = A.flattened_fwd_bwd(s.cu_prompt, s.cu_branch, s.cu_resp, 4, 2, s.scale,
                              qp, kp, vp, qr, kr, vr, dop, dor)
    for g in range(s.num_groups):
        p0, p1 = s.cu_prompt[g], s.cu_prompt[g + 1]
        P = p1 - p0
        pos = np.arange(P)
        assert np.max(np.abs(out["lse_p"][:, p0:p1] - np.log(pos + 1))) < 1e-14
        assert np.max(np.abs(out["o_p"][p0:p1, :, 0] - (pos / 2)[:, None])) < 1e-12
        for b in range(s.cu_branch[g], s.cu_branch[g + 1]):
            r0, r1 = s.cu_resp[b], s.cu_resp[b + 1]
            t = np.arange(r1 - r0)
            assert np.max(np.abs(out["lse_r"][:, r0:r1] - np.log(P + t + 1))) < 1e-14
            assert np.max(np.abs(out["o_r"][r0:r1, :, 0] - ((P + t) / 2)[:, None])) < 1e-12


def test_pool_matches_serial():
    gi = I.make_inputs(SMALL, seed=18)
    a = run(A.flattened_fwd_bwd, gi)
    b = run(A.flattened_fwd_bwd, gi, workers=3)
    for k in a:
        assert np.array_equal(a[k], b[k]), k


# --------------------------------------------------------------------------- sampled rows

def test_sampled_rows_match_flattened():
    s = SMALL
    gi = I.make_inputs(s, seed=19, qk_mult=1.0)
    fl = run(A.flattened_fwd_bwd, gi)

    class T:
        pass
    t = T()
    t.cu_prompt, t.cu_branch, t.cu_resp = s.cu_prompt, s.cu_branch, s.cu_resp
    t.num_q_heads, t.num_kv_heads, t.head_dim = 4, 2, 16
    for name in ("q_p", "k_p", "v_p", "q_r", "k_r", "v_r", "do_p", "do_r"):
        setattr(t, name, getattr(gi, name))
    for h in (0, 3):
        rows = [0, 5, 12, 13, 18]
        got = S.query_rows(t, "prompt", rows, h)
        assert rel(got["o"], fl["o_p"][rows, h]) < 1e-12
        assert np.max(np.abs(got["lse"] - fl["lse_p"][h, rows])) < 1e-12
        assert rel(got["dq"], fl["dq_p"][rows, h]) < 1e-12
        rows = [0, 8, 9, 12, 20, 28]
        got = S.query_rows(t, "resp", rows, h)
        assert rel(got["o"], fl["o_r"][rows, h]) < 1e-12
        assert np.max(np.abs(got["lse"] - fl["lse_r"][h, rows])) < 1e-12
        assert rel(got["dq"], fl["dq_r"][rows, h]) < 1e-12
    for kh in (0, 1):
        for rows in ([0, 4, 12], [13, 17, 18]):
            got = S.key_rows(t, "prompt", rows, kh)
            assert rel(got["dk"], fl["dk_p"][rows, kh]) < 1e-12
            assert rel(got["dv"], fl["dv_p"][rows, kh]) < 1e-12
        for rows in ([0, 3, 8], [12, 13, 15], [27]):
            got = S.key_rows(t, "resp", rows, kh)
            assert rel(got["dk"], fl["dk_r"][rows, kh]) < 1e-12
            assert rel(got["dv"], fl["dv_r"][rows, kh]) < 1e-12


def test_sampled_key_rows_pool_matches_serial():
    """The pooled key-row reference adds the same terms in the same order as
    the serial one: identical bits."""
    s = SMALL
    gi = I.make_inputs(s, seed=20, qk_mult=1.0)

    class T:
        pass
    t = T()
    t.cu_prompt, t.cu_branch, t.cu_resp = s.cu_prompt, s.cu_branch, s.cu_resp
    t.num_q_heads, t.num_kv_heads, t.head_dim = 4, 2, 16
    for name in ("q_p", "k_p", "v_p", "q_r", "k_r", "v_r", "do_p", "do_r"):
        setattr(t, name, getattr(gi, name))
    for kind, rows in (("prompt", [0, 4, 12]), ("prompt", [13, 17, 18]), ("resp", [12, 13, 15])):
        a = S.key_rows(t, kind, rows, 1)
        b = S.key_rows(t, kind, rows, 1, workers=3)
        assert np.array_equal(a["dk"], b["dk"]) and np.array_equal(a["dv"], b["dv"])


# --------------------------------------------------------------------------- golden regression

def test_golden_tiny_fixture():
    import json
    import os
    import sys
    sys.path.insert(0, os.path.join(os.path.dirname(__file__), "golden"))
    import make_golden
    with open(os.path.join(os.path.dirname(__file__), "golden", "tiny_oracle.json")) as f:
        doc = json.load(f)
    out = make_golden.compute()
    for k, v in doc["norms"].items():
        assert abs(np.linalg.norm(out[k]) - v) <= 1e-12 * max(v, 1.0), k
    for k, ents in doc["entries"].items():
        for ix, val in ents:
            assert abs(out[k][tuple(ix)] - val) <= 1e-12 * max(abs(val), 1.0), (k, ix)
