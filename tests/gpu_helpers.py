"""Shared helpers of the GPU parity tests: run the HIP path through the C ABI
and compare with the fp64 oracle at the stated tolerances.

Tolerances (relative Frobenius error per tensor, LSE max absolute error):
O <= 1e-2, LSE <= 1e-3, dQ/dK/dV (prompt gradients included) <= 2e-2.
"""
import numpy as np
import torch

from oracle import attention as A
from paper_2609_33133_amd import inputs as I
from paper_2609_33133_amd.api import GroupBatch, REPLAY_FUSED
from paper_2609_33133_amd.group_attention import FlattenedStep, SharedStep, upload

TOL_O = 1e-2
TOL_LSE = 1e-3
TOL_GRAD = 2e-2
O_KEYS = ("o_p", "o_r")
LSE_KEYS = ("lse_p", "lse_r")
GRAD_KEYS = ("dq_p", "dk_p", "dv_p", "dq_r", "dk_r", "dv_r")


def log(msg):
    print(msg, flush=True)


def to_np(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def run_shared(gi, mode=REPLAY_FUSED, n_seed=None, device="cuda", path="tree"):
    """The method's step through the C ABI: path "tree" (augtree_tree_fwd +
    augtree_tree_bwd) or "calls" (the six separate entry points)."""
    b = GroupBatch.from_shape(gi.shape)
    step = SharedStep(b, device, mode=mode, n_seed=n_seed, path=path)
    x = upload(gi, device)
    step.run(x)
    torch.cuda.synchronize()
    return {k: to_np(v) for k, v in step.outputs().items()}, step


def run_flattened(gi, device="cuda"):
    b = GroupBatch.from_shape(gi.shape)
    step = FlattenedStep(b, device)
    x = upload(gi, device)
    step.materialize(x)
    step.run()
    torch.cuda.synchronize()
    return {k: to_np(v) for k, v in step.outputs().items()}


def oracle(gi, workers=1):
    s = gi.shape
    c = I.bf16_bits_to_f64
    return A.flattened_fwd_bwd(s.cu_prompt, s.cu_branch, s.cu_resp, s.num_q_heads, s.num_kv_heads, s.scale,
                               *(c(getattr(gi, n)) for n in ("q_p", "k_p", "v_p", "q_r", "k_r", "v_r", "do_p",
                                                             "do_r")), workers=workers)


def rel(a, b):
    nb = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / (nb if nb > 0 else 1.0))


def errors(got, ref):
    e = {}
    for k in O_KEYS + GRAD_KEYS:
        e[k] = rel(got[k], ref[k])
    for k in LSE_KEYS:
        e[k] = float(np.max(np.abs(got[k] - ref[k])))
    return e


def assert_close(got, ref, label=""):
    e = errors(got, ref)
    log(f"[{label}] " + " ".join(f"{k}={v:.2e}" for k, v in e.items()))
    bad = [k for k in O_KEYS if not e[k] <= TOL_O]
    bad += [k for k in LSE_KEYS if not e[k] <= TOL_LSE]
    bad += [k for k in GRAD_KEYS if not e[k] <= TOL_GRAD]
    assert not bad, f"{label}: out of tolerance: {[(k, e[k]) for k in bad]}"
    return e
