"""Writes tests/golden/layer_c3_8x8_b1_k3_tl.json from the CPU oracle only.

The 8x8, 3-channel, k = 3, TL-padded single-image workload with the seeded
inputs of paper_2301_09266_amd.synth: x, K, y = forward(x), log|det|, and the
inverse of z.  Re-run after a justified change to the oracle:
    python tests/golden/make_golden.py
"""
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_2301_09266_amd import synth  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "layer_c3_8x8_b1_k3_tl.json")


def main():
    o = oracle.default()
    c = synth.make("layer_c3_8x8_b1_k3")
    y = o.forward(c["x"], c["K"], 0)
    rec = dict(
        source="oracle/finc_oracle.c via tests/golden/make_golden.py",
        workload="layer_c3_8x8_b1_k3 (TL padding)",
        x=c["x"].ravel().tolist(), K=c["K"].ravel().tolist(),
        y=y.ravel().tolist(), logdet=o.logdet(c["K"], 0, 8, 8),
        z=c["z"].ravel().tolist(), inv_z=o.inverse(c["z"], c["K"], 0).ravel().tolist(),
    )
    with open(OUT, "w") as f:
        json.dump(rec, f, indent=0)
        f.write("\n")


if __name__ == "__main__":
    main()
