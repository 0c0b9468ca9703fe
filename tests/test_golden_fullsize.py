"""The stored full-size oracle results (tests/golden/fullsize_<key>.npz) are
consistent with what they claim, CPU only: the oracle's restore reproduced its
never-evicted prefill at full size (both restore invariants: recomputed K/V
equal to the clean prefill's, first-token logits equal to the never-evicted
ones), the restore's row counts are those of the row-set definition for the
workload's plan, every sampled K/V position is a row written at its layer in
its chunk, and the stored token is the stored logits' argmax with the stored
top-2 margin."""

import os

import numpy as np
import pytest

import oracle as O
from paper_2609_01338_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.mark.parametrize("key", ["1b", "3b", "1p5b", "8b"])
def test_golden_consistent(key):
    path = os.path.join(GOLDEN, f"fullsize_{key}.npz")
    if not os.path.exists(path):
        pytest.skip(f"{path} not written yet")
    g = np.load(path)
    w = W.WORKLOADS[key]
    C = w.model.chunk_tokens
    plan = W.make_plan(w)
    assert float(g["logits_vs_clean"]) <= 1e-9 and float(g["kv_vs_clean"]) == 0.0
    assert int(g["clean_token"]) == int(g["token"])
    R, D = O.restore_rows(plan.kv_state, w.n_ctx, w.n_prompt, C)
    assert g["nR"].tolist() == [r.size for r in R] and g["nD"].tolist() == [d.size for d in D]
    for l, c, p in zip(g["kv_layer"], g["kv_chunk"], g["kv_pos"]):
        assert p // C == c and p in set(D[l][D[l] // C == c].tolist())
    # one sampled row per (layer, chunk) holding a written row, no more
    want = sum(np.unique(d // C).size for d in D)
    assert g["kv_layer"].size == want
    assert g["k"].shape == g["v"].shape == (want, w.model.dkv) and g["k"].dtype == np.float16
    lg = g["logits"].astype(np.float64)
    assert lg.shape == (w.model.vocab,) and int(np.argmax(lg)) == int(g["token"])
    top = np.sort(lg)[-2:]
    assert abs((top[1] - top[0]) - float(g["margin"])) <= 1e-5 * max(1.0, abs(top[1]))
