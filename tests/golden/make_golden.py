"""Writes tests/golden/tiny_oracle.txt from the CPU oracle alone.

The paper prints no worked example for the hot path (no scores, kept sets or
attention outputs), so this fixture is not a paper value: it freezes what the
pinned oracle computes on the tiny 2-head fp32 workload (seed 0) so that a
later change to the oracle's arithmetic shows up as a diff.  Run:

    python tests/golden/make_golden.py
"""
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle  # noqa: E402
import workloads as W  # noqa: E402

ROWS = [0, 1, 17, 33, 63]


def main(path=os.path.join(HERE, "tiny_oracle.txt")):
    cfg = W.tiny_config()
    x = W.make_layer_inputs(cfg, seed=0)
    r = oracle.run_layer(cfg, x, rows=np.array(ROWS, np.int32))
    with open(path, "w") as f:
        f.write("# oracle output, tiny fp32 workload (2 heads, d=64, F=64, H=4, L=64), seed 0\n")
        f.write("# written by tests/golden/make_golden.py (calls oracle/ only)\n")
        for h in range(cfg.n_heads):
            f.write(f"head {h} kv_len {int(r.kv_len[h])}\n")
            f.write("kept " + " ".join(str(int(v)) for v in r.kept_seg[h]) + "\n")
            f.write("scores_hex " + " ".join(f"{int(v):08x}" for v in r.scores[h].view(np.uint32)) + "\n")
            for i, row in enumerate(ROWS):
                f.write(f"row {row} lse {r.lse[h, i]:.17g} o " + " ".join(f"{v:.17g}" for v in r.O[h, i]) + "\n")


if __name__ == "__main__":
    main()
