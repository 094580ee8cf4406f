"""Write the oracle regression fixtures in this folder.

The paper prints no worked numerical example for Eq. (10), so these fixtures
are not the paper's numbers: they freeze the fp64 oracle's output on the
smallest synthetic workload (one head, n = 128, d = 64, m = 64) so that any
later change to the oracle's arithmetic shows up as a diff.  Only ``oracle``
and the input generator are called here.

    python tests/golden/make_golden.py
"""
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle  # noqa: E402
from paper_2106_12566_amd import synth  # noqa: E402

ROWS = [0, 1, 2, 63, 64, 100, 127]


def main():
    d = synth.make(1)
    z, den = oracle.attention(d["q"], d["k"], d["v"], d["b"], d["W"])
    out = {
        "what": "Eq. (10) evaluated by the fp64 oracle on workload 1 (B=1, H=1, n=128, d=64, m=64)",
        "generator": "paper_2106_12566_amd.synth.make(1)",
        "rows": ROWS,
        "z": [[float(x) for x in z[0, 0, i]] for i in ROWS],
        "den": [float(den[0, 0, i]) for i in ROWS],
    }
    with open(os.path.join(HERE, "tiny_n128_rows.json"), "w") as f:
        json.dump(out, f, indent=1)


if __name__ == "__main__":
    main()
