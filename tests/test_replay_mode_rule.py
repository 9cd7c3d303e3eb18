"""The per-group replay-forward mode rule (AUGTREE_REPLAY_AUTO): host logic
only, no GPU. Its decisions on shapes whose two modes were timed on an
MI355X (replay_fwd alone, Hq=32, Hkv=8, d=128) agree with the faster mode
wherever the two differ by more than 10 %:

    P      G   R      fused ms  split ms
    32768  16  16     1.035     0.645
    32768  16  64     1.080     0.719
    32768  16  128    1.183     1.077
    8192   64  8      1.002     0.201
    8192   64  32     1.033     0.320
    8192   64  200    2.147     1.877
    4096   8   4096   3.272     3.535

(32768, 16, 128) is a near tie the rule prices equal (16 full tiles x 514
blocks either way) and gives to FUSED for the merge; SPLIT measured 9 %
faster there.
"""
import numpy as np
import pytest

from paper_2609_33133_amd import api
from paper_2609_33133_amd import inputs as I
from paper_2609_33133_amd.api import GroupBatch

TIMED = [((32768, 16, 16), 1), ((32768, 16, 64), 1), ((8192, 64, 8), 1),
         ((8192, 64, 32), 1), ((8192, 64, 200), 1), ((4096, 8, 4096), 0)]


@pytest.mark.parametrize("shape,split", TIMED)
def test_rule_matches_timed_winner(shape, split):
    P, G, R = shape
    b = GroupBatch.from_shape(I.custom_shape([P], [[R] * G], 32, 8, 128))
    assert api.replay_split_groups(b).tolist() == [split]


def test_rule_is_per_group():
    s = I.custom_shape([4096, 32768, 2048], [[4096] * 8, [16] * 16, [3000, 1]], 32, 8, 128)
    got = api.replay_split_groups(GroupBatch.from_shape(s)).tolist()
    assert got[:2] == [0, 1]
    assert got[2] in (0, 1)


def test_workloads_stay_fused():
    # the headline workloads' branches are long: the rule keeps them fused
    for name in ("balanced", "prompt", "response"):
        b = GroupBatch.from_shape(I.config_shape(name))
        assert not api.replay_split_groups(b).any(), name


def test_bad_descriptor_reported():
    b = GroupBatch(np.array([0, 5], np.int32), np.array([0, 1], np.int32), np.array([0, 0], np.int32), 2, 1, 64)
    with pytest.raises(Exception):
        api.replay_split_groups(b)
