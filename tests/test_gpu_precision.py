"""Keys with a large shared component: the dQ product takes dS rounded to
bf16, and sum_j dS~_j k_j multiplies the rounding error of dS~ by the shared
part of the keys while dQ itself only sees their differences (every row of
dS sums to zero over its keys). The dQ kernel subtracts c * sum_j dS~_j with
c the mean of the group's first 64 prompt keys, which removes a shared
component that is the same for every key; a component that varies along the
positions (a ramp) is only reduced to its variation over the keys that carry
the softmax mass. Both cases against the fp64 oracle, with the errors
measured on the GPU written into the bounds."""
import numpy as np
import pytest
import torch

from paper_2609_33133_amd import inputs as I
from paper_2609_33133_amd.api import REPLAY_FUSED, REPLAY_SPLIT

from gpu_helpers import TOL_GRAD, assert_close, errors, log, oracle, run_shared

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _biased_keys(seed, norm):
    """Keys N(0,1)/sqrt(d) plus one bias vector per KV head of norm `norm`
    (the same for every prompt and response key of the head)."""
    shape = I.custom_shape([300, 70], [[200, 77, 129], [1, 64]], 8, 2, 128)
    gi = I.make_inputs(shape, seed=seed, qk_mult=1.0)
    rng = np.random.default_rng(seed)
    bias = rng.standard_normal((2, 128)).astype(np.float32)
    bias *= norm / np.linalg.norm(bias, axis=1, keepdims=True)
    for name in ("k_p", "k_r"):
        k = I.bf16_bits_to_f32(getattr(gi, name)) + bias[None]
        setattr(gi, name, I.f32_to_bf16_bits(k))
    return gi


@pytest.mark.parametrize("norm", [8.0, 64.0])
def test_key_bias_does_not_amplify_dq_error(norm):
    """A bias of norm 8 or 64 on every key (the random part has norm ~1):
    uncorrected, the dQ error grows with the bias (at norm 64 past the 2e-2
    tolerance); with the correction every tensor stays at the unbiased
    level."""
    gi = _biased_keys(61, norm)
    ref = oracle(gi)
    for mode, path in ((REPLAY_FUSED, "tree"), (REPLAY_SPLIT, "calls")):
        got, _ = run_shared(gi, mode=mode, path=path)
        e = assert_close(got, ref, f"key bias {norm} {path}")
        assert e["dq_p"] < 5e-3 and e["dq_r"] < 5e-3, e


def _steep_ramp():
    """Logits rising along the key positions (as in the parity test with the
    rising logits) but with the ramp carried by a 10x steeper key component
    k[0] = j / 64 and 10x flatter query slopes: the keys that carry the
    softmax mass share a large, position-dependent k[0] (up to ~15 against a
    random part of norm ~0.1)."""
    shape = I.custom_shape([700], [[150, 90]], 8, 2, 128)
    gi = I.make_inputs(shape, seed=11)
    P = shape.prompt_lens[0]
    slopes = np.array([0.0, 40.0, 160.0, 400.0, 640.0, 1000.0, 1570.0, -300.0], np.float32) / 10
    gi.q_p[:, :, 0] = I.f32_to_bf16_bits(np.broadcast_to(slopes, (P, 8)).copy())
    gi.q_r[:, :, 0] = I.f32_to_bf16_bits(np.broadcast_to(slopes, (gi.q_r.shape[0], 8)).copy())
    gi.k_p[:, :, 0] = I.f32_to_bf16_bits((np.arange(P, dtype=np.float32) / 64)[:, None].repeat(2, 1))
    for b in range(2):
        r0, r1 = shape.cu_resp[b], shape.cu_resp[b + 1]
        pos = (P + np.arange(r1 - r0, dtype=np.float32)) / 64
        gi.k_r[r0:r1, :, 0] = I.f32_to_bf16_bits(pos[:, None].repeat(2, 1))
    return gi


# measured on an MI355X: dQ_P 1.50e-2, dQ_R 2.80e-2 (every other tensor <= 2.6e-3); bound with margin
RAMP_DQ_BOUND = 4e-2


def test_steep_key_ramp_dq_error_bound():
    """The recorded limit: on the steep ramp the dQ error exceeds the 2e-2
    tolerance (a position-dependent shared key component is not removed by
    one correction vector); every other tensor is within tolerance, and dQ
    stays under the recorded bound."""
    gi = _steep_ramp()
    ref = oracle(gi)
    for mode, path in ((REPLAY_FUSED, "tree"), (REPLAY_FUSED, "calls")):
        got, _ = run_shared(gi, mode=mode, path=path)
        e = errors(got, ref)
        log(f"[steep ramp {path}] " + " ".join(f"{k}={v:.2e}" for k, v in e.items()))
        for k in ("o_p", "o_r"):
            assert e[k] <= 1e-2, k
        for k in ("lse_p", "lse_r"):
            assert e[k] <= 1e-3, k
        for k in ("dk_p", "dv_p", "dk_r", "dv_r"):
            assert e[k] <= TOL_GRAD, k
        assert e["dq_p"] <= RAMP_DQ_BOUND and e["dq_r"] <= RAMP_DQ_BOUND, e
