"""The autograd op over the C ABI (group_attention): outputs and the
gradients torch.autograd returns for L = sum(dO_P * O_P) + sum(dO_R * O_R)
against the fp64 oracle, and bitwise against the explicit step."""
import numpy as np
import pytest
import torch

from paper_2609_33133_amd import inputs as I
from paper_2609_33133_amd.api import REPLAY_FUSED, REPLAY_SPLIT, GroupBatch
from paper_2609_33133_amd.autograd import group_attention
from paper_2609_33133_amd.group_attention import SharedStep, upload

from gpu_helpers import assert_close, oracle, to_np

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _leaves(x):
    return {n: x[n].clone().requires_grad_(True) for n in ("q_p", "k_p", "v_p", "q_r", "k_r", "v_r")}


def _run(gi, mode, zero_do_p=False):
    b = GroupBatch.from_shape(gi.shape)
    x = upload(gi, "cuda")
    leaf = _leaves(x)
    o_p, o_r = group_attention(leaf["q_p"], leaf["k_p"], leaf["v_p"], leaf["q_r"], leaf["k_r"], leaf["v_r"], b,
                               mode=mode)
    loss = (o_r.float() * x["do_r"].float()).sum()
    if not zero_do_p:
        loss = loss + (o_p.float() * x["do_p"].float()).sum()
    loss.backward()
    torch.cuda.synchronize()
    got = {"o_p": to_np(o_p), "o_r": to_np(o_r)}
    for n in ("q_p", "k_p", "v_p", "q_r", "k_r", "v_r"):
        got["d" + n] = to_np(leaf[n].grad)
    return got, b, x


@pytest.mark.parametrize("mode", [REPLAY_FUSED, REPLAY_SPLIT])
def test_autograd_matches_oracle(mode):
    shape = I.custom_shape([300, 70], [[200, 77, 129], [1, 64]], 8, 2, 128)
    gi = I.make_inputs(shape, seed=31)
    got, _, _ = _run(gi, mode)
    ref = oracle(gi)
    # LSE is not an output of the op: compare it as the oracle's own value
    got["lse_p"], got["lse_r"] = ref["lse_p"], ref["lse_r"]
    assert_close(got, ref, f"autograd mode={mode}")


def test_autograd_equals_explicit_step_bitwise():
    gi = I.make_config("tiny")
    got, b, x = _run(gi, REPLAY_FUSED)
    step = SharedStep(b, "cuda", mode=REPLAY_FUSED)
    step.run(x)
    torch.cuda.synchronize()
    out = {k: to_np(v) for k, v in step.outputs().items()}
    for k in ("o_p", "o_r", "dq_p", "dk_p", "dv_p", "dq_r", "dk_r", "dv_r"):
        assert np.array_equal(got[k], out[k]), k


def test_autograd_unused_prompt_output():
    """Only O_R reaches the loss: the prompt rows get no upstream gradient,
    which the oracle reproduces with dO_P = 0."""
    shape = I.custom_shape([150], [[40, 90, 7]], 4, 2, 64)
    gi = I.make_inputs(shape, seed=32)
    got, _, _ = _run(gi, REPLAY_FUSED, zero_do_p=True)
    gi.do_p = np.zeros_like(gi.do_p)
    ref = oracle(gi)
    got["lse_p"], got["lse_r"] = ref["lse_p"], ref["lse_r"]
    assert_close(got, ref, "autograd dO_P = 0")
