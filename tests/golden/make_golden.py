"""Writes tests/golden/tiny_oracle.json from the fp64 oracle alone.

Workload: the tiny replay tree (1 group, P=256, G=2 branches of R=128, Hq=Hkv=4,
d=64, seed 0). Stored: summary norms of every output and a few individual
entries. The paper prints no worked numeric example, so these values come only
from oracle/attention.py (the flattened definition of §2.1-§2.2) and pin it
against accidental change. Run: python tests/golden/make_golden.py
"""
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import attention as A  # noqa: E402
from paper_2609_33133_amd import inputs as I  # noqa: E402

PICKS = {"o_p": [(0, 0, 0), (255, 3, 63), (100, 1, 7)], "o_r": [(0, 0, 0), (255, 2, 5), (127, 1, 9)],
         "lse_p": [(0, 0), (3, 255)], "lse_r": [(0, 0), (2, 200)],
         "dq_p": [(17, 2, 3)], "dk_p": [(0, 0, 0), (255, 3, 1)], "dv_p": [(128, 1, 60)],
         "dq_r": [(129, 3, 0)], "dk_r": [(5, 2, 2)], "dv_r": [(255, 0, 31)]}


def compute():
    gi = I.make_config("tiny")
    s = gi.shape
    c = I.bf16_bits_to_f64
    return A.flattened_fwd_bwd(s.cu_prompt, s.cu_branch, s.cu_resp, s.num_q_heads, s.num_kv_heads, s.scale,
                               *(c(x) for x in (gi.q_p, gi.k_p, gi.v_p, gi.q_r, gi.k_r, gi.v_r, gi.do_p, gi.do_r)))


def main():
    out = compute()
    doc = {"workload": "tiny: P=256, G=2, R=128, Hq=Hkv=4, d=64, seed 0",
           "source": "oracle/attention.py flattened_fwd_bwd",
           "norms": {k: float(np.linalg.norm(v)) for k, v in out.items()},
           "entries": {k: [[list(ix), float(out[k][ix])] for ix in v] for k, v in PICKS.items()}}
    with open(os.path.join(os.path.dirname(__file__), "tiny_oracle.json"), "w") as f:
        json.dump(doc, f, indent=1)


if __name__ == "__main__":
    main()
