"""Writes tests/golden/rounding_attribution.txt: for a workload's model, the
per-layer max |K, V| distance between an fp64 prefill of the first 64 context
tokens and prefills whose matrix-product operands are rounded in different
ways (oracle/f16_floor.py): which rounding moves the stored keys and values,
and by how much, over the model's depth.  Calls only oracle/ and the seeded
input generator.

    python tests/golden/make_rounding_attribution.py [--threads T] [keys...]
"""

import argparse
import os
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import oracle as O  # noqa: E402
from oracle.f16_floor import EXACT, Rounding, kv_distance, prefix_kv  # noqa: E402
from paper_2609_01338_amd import workloads as W  # noqa: E402

N_PREFIX = 64
OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "rounding_attribution.txt")

# (name, weights, activations, attention probabilities)
VARIANTS = [
    ("half-operands", Rounding("half", "half", "exact")),      # the half-operand floor
    ("half-operands+P", Rounding("half", "half", "half")),     # plus P in half before P.V
    ("exact-weights+half-acts+P", Rounding("exact", "half", "half")),
    ("exact-weights+half-acts", Rounding("exact", "half", "exact")),
    ("half-weights+exact-acts", Rounding("half", "exact", "exact")),
    ("P-only", Rounding("exact", "exact", "half")),
    ("bf16-operands+P", Rounding("bf16", "bf16", "bf16")),
]


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--threads", type=int, default=4)
    ap.add_argument("keys", nargs="*", default=["8b", "3b"])
    a = ap.parse_args()
    lines = [f"# per-layer max |K,V(rounded operands) - K,V(fp64)| over the first {N_PREFIX} context tokens",
             "# written by tests/golden/make_rounding_attribution.py (oracle/ and the input generator only)",
             "# rounding = weights/activations/attention-probabilities, each exact, half or bf16",
             "# key variant n_layers max d_l0 d_l1 ..."]
    for key in a.keys:
        w = W.WORKLOADS[key]
        hp = O.Hyper(w.model)
        wts = O.Weights(hp, W.make_blob(w), threads=a.threads)
        ctx, _ = W.make_tokens(w)
        toks = ctx[:N_PREFIX]
        t = time.time()
        K0, V0, _ = prefix_kv(hp, wts, toks, EXACT)
        for name, r in VARIANTS:
            K1, V1, _ = prefix_kv(hp, wts, toks, r)
            d = kv_distance((K1, V1), (K0, V0))
            lines.append(f"{key} {name} {hp.n_layers} {d.max():.6e} " + " ".join(f"{x:.6e}" for x in d))
            print(f"{key} {name}: max {d.max():.3e} layer0 {d[0]:.3e} ({time.time() - t:.0f} s)", flush=True)
    with open(OUT, "w") as f:
        f.write("\n".join(lines) + "\n")


if __name__ == "__main__":
    main()
