"""Writes tests/golden/tiny_oracle.json from the fp64 oracle alone.

The paper prints no worked numeric example (its figures report error and
memory curves only), so this fixture is a regression pin of the oracle on the
tiny workload (B=1, L=1024, D=16, N=16, K=1, dx = unit impulse at t=0, d=0),
not a value from the paper.  It calls only oracle/ and the seeded input
module.  Run from the repository root:  python tests/golden/make_golden.py
"""
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import oracle                       # noqa: E402
from paper_2512_23068_amd import inputs         # noqa: E402


def main():
    inp = inputs.make_inputs("tiny")
    y, dy, _, _ = oracle.scan_jvp(inp["x"], inp["dx"], inp)
    pts = [(0, 0), (0, 5), (1, 0), (3, 15), (17, 7), (100, 2), (511, 11), (777, 0), (1023, 9), (1023, 0)]
    samples = [[t, d, float(y[0, t, d]), float(dy[0, 0, t, d])] for (t, d) in pts]
    out = {"workload": "tiny (B=1,L=1024,D=16,N=16,K=1)", "source": "fp64 oracle (oracle/pgf_oracle.c)",
           "samples": samples}
    with open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "tiny_oracle.json"), "w") as f:
        json.dump(out, f, indent=1)


if __name__ == "__main__":
    main()
