"""The autograd op has no CPU path: host tensors are refused before any
library call (CPU only)."""
import pytest
import torch

from paper_2609_33133_amd import inputs as I
from paper_2609_33133_amd.api import GroupBatch
from paper_2609_33133_amd.autograd import group_attention


def test_refuses_host_tensors():
    s = I.custom_shape([5], [[3, 2]], 2, 1, 64)
    b = GroupBatch.from_shape(s)
    bf = torch.bfloat16
    q_p = torch.zeros((5, 2, 64), dtype=bf, requires_grad=True)
    kv_p = torch.zeros((5, 1, 64), dtype=bf)
    q_r = torch.zeros((5, 2, 64), dtype=bf)
    kv_r = torch.zeros((5, 1, 64), dtype=bf)
    with pytest.raises(ValueError, match="no CPU path"):
        group_attention(q_p, kv_p, kv_p, q_r, kv_r, kv_r, b)
