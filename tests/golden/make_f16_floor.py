"""Writes tests/golden/f16_operand_floor.txt: for each workload, the per-layer
max |K, V| distance between an fp64 prefill and a half-operand prefill of the
first 64 context tokens (oracle/f16_floor.py).  Calls only oracle/ and the
seeded input generator.

    python tests/golden/make_f16_floor.py [keys...]
"""

import os
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import oracle as O  # noqa: E402
from oracle.f16_floor import f16_operand_floor  # noqa: E402
from paper_2609_01338_amd import workloads as W  # noqa: E402

N_PREFIX = 64
OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "f16_operand_floor.txt")


def main():
    keys = sys.argv[1:] or ["1b", "3b", "1p5b", "8b"]
    lines = [f"# per-layer max |K,V(half operands) - K,V(fp64)| over the first {N_PREFIX} context tokens",
             "# written by tests/golden/make_f16_floor.py (oracle/ and the input generator only)",
             "# key n_layers floor_l0 floor_l1 ..."]
    for key in keys:
        w = W.WORKLOADS[key]
        t = time.time()
        hp = O.Hyper(w.model)
        wts = O.Weights(hp, W.make_blob(w))
        ctx, _ = W.make_tokens(w)
        fl = f16_operand_floor(hp, wts, ctx[:N_PREFIX],
                               lambda run, l: print(f"{key} {run} layer {l}", flush=True) if l % 8 == 7 else None)
        lines.append(f"{key} {w.model.n_layers} " + " ".join(f"{x:.6e}" for x in fl))
        print(f"{key}: max floor {fl.max():.3e} ({time.time() - t:.0f} s)", flush=True)
    with open(OUT, "w") as f:
        f.write("\n".join(lines) + "\n")


if __name__ == "__main__":
    main()
