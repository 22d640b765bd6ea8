"""Write the oracle regression fixture for the smallest workload.

Provenance: every value in the fixture is produced by ``oracle/`` alone on the
seeded inputs of ``paper_2608_17379_amd.workloads`` (B=1, H=1, S=128, D=64,
non-causal, scale 1/8, seed 0).  The paper prints no worked numeric example,
so this file pins nothing by itself; it guards the oracle (already pinned by
tests/test_oracle.py) against unnoticed later changes.

    python tests/golden/make_golden.py
"""
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle  # noqa: E402
from paper_2608_17379_amd import workloads as wl  # noqa: E402

ROWS = [0, 1, 63, 64, 127]


def main():
    w = wl.WORKLOADS["mha_b1_h1_s128_d64"]
    x = wl.make_inputs(w, 0)
    o, lse = oracle.attention_forward(x.q, x.k, x.v, w.causal, w.scale)
    dq, dk, dv = oracle.attention_backward(x.q, x.k, x.v, x.do, w.causal, w.scale)
    fx = {
        "workload": w.name, "seed": 0, "rows": ROWS,
        "lse_rows": [float(lse[0, 0, i]) for i in ROWS],
        "o_rows_first8": [[float(t) for t in o[0, 0, i, :8]] for i in ROWS],
        "norms": {n: float(t.norm()) for n, t in
                  (("o", o), ("dq", dq), ("dk", dk), ("dv", dv))},
        "sums": {n: float(t.sum()) for n, t in
                 (("o", o), ("lse", lse), ("dq", dq), ("dk", dk), ("dv", dv))},
    }
    with open(os.path.join(HERE, "oracle_mha_b1_h1_s128_d64_seed0.json"), "w") as f:
        json.dump(fx, f, indent=1)
        f.write("\n")


if __name__ == "__main__":
    main()
