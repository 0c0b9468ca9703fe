"""Full-size restore on the GPU, in the configuration the benchmark times.

For every workload at its full shape (all layers, full context and prompt,
its own eviction plan):
 * the first token after evict -> restore equals that of a never-evicted
   prefill of the same tokens (or is a near-tie of it) and every first-token
   logit is within 5e-2 of it.  Not bit for bit: the restore runs the prompt
   rows alone through projections of a few rows, which are split over K
   (and their attention over keys), so their fp32 sums are added in another
   order than inside the prefill's full-height GEMMs;
 * sampled (layer, chunk) K/V slots of the cached context read back after
   the restore: swapped (restored bytes) and resident (untouched) slots are
   byte-identical to the same slots before the eviction; recomputed slots
   agree with them within twice the oracle K/V tolerance below (each side
   is within that tolerance of the exact values; the recompute may take
   split paths where it carries few rows of a layer);
 * the first 64 positions of every layer match the CPU oracle's prefill of
   the first 64 context tokens (causality makes those rows independent of the
   rest of the context): K/V within max(2e-2, 1.25 x the half-operand floor
   of this model, tests/golden/f16_operand_floor.txt) -- the accumulated
   rounding of half-precision matrix operands over 28-32 layers exceeds 2e-2
   on its own -- and, for a 64-token context run through all layers on the
   GPU, first-token logits within 5e-2 and the same greedy token (near-tie
   rule as in the end-to-end tests).
"""

import os

import numpy as np
import pytest

import oracle as O
from paper_2609_01338_amd import mz
from paper_2609_01338_amd import workloads as W
from gpu_util import report, torch_cuda

pytestmark = pytest.mark.gpu

KV_TOL = 2e-2
LOGIT_TOL = 5e-2
FLOOR_MARGIN = 1.25
N_ORACLE = 64


def _floor(key):
    """Max over layers of the stored half-operand floor for this workload."""
    path = os.path.join(os.path.dirname(__file__), "golden", "f16_operand_floor.txt")
    with open(path) as f:
        for line in f:
            parts = line.split()
            if parts and parts[0] == key:
                return max(float(x) for x in parts[2:])
    raise KeyError(key)


def _oracle_prefix(m, blob, tokens):
    """Oracle K/V (float64 [L][n, dkv]) of a prefill over `tokens`, and its
    first-token logits."""
    hp = O.Hyper(m)
    wts = O.Weights(hp, blob)
    n = tokens.size
    pos = np.arange(n)
    h = wts.rows("emb", tokens.astype(np.int64))
    Ks, Vs = [], []
    for l in range(m.n_layers):
        K = np.zeros((n, m.dkv), np.float16)
        V = np.zeros((n, m.dkv), np.float16)

        def write(k, v, K=K, V=V):
            K[:], V[:] = k, v

        def read(last, K=K, V=V):
            return K[:last].astype(np.float64), V[:last].astype(np.float64)

        h = O.layer_forward(hp, wts.layer(l), h, pos, write, read)
        Ks.append(K.astype(np.float64))
        Vs.append(V.astype(np.float64))
        if l % 8 == 7:
            report("  oracle prefix", layers_done=l + 1)
    return Ks, Vs, O.output_logits(hp, wts, h[-1])


@pytest.mark.parametrize("key", ["1b", "3b", "1p5b", "8b"])
def test_full_size_restore(key):
    torch_cuda()
    w = W.WORKLOADS[key]
    m = w.model
    L, C, dkv = m.n_layers, m.chunk_tokens, m.dkv
    S = w.n_ctx + w.n_prompt
    nc = w.n_chunks
    report("full size", workload=key, layers=L, n_ctx=w.n_ctx, n_prompt=w.n_prompt)
    blob = W.make_blob(w)
    ctx, prompt = W.make_tokens(w)
    plan = W.make_plan(w)
    eng = mz.Engine(m, blob, max_ctx=S)
    try:
        e = eng.ctx
        mz.mz_prefill_context(e, np.concatenate([ctx, prompt]))
        clean_tok, clean_logits = mz.mz_first_token(e, m.vocab)
        mz.mz_truncate_context(e, w.n_ctx)
        layers = sorted({0, L // 2, L - 1})
        chunks = sorted({0, nc // 2, nc - 1})
        pre = {(l, c): mz.mz_read_kv(e, l, c, C, dkv) for l in layers for c in chunks}
        report("  plan", **plan.counts(), weight_units_swapped=int((plan.w_state == W.SWAP).sum()))
        mz.mz_evict(e, plan.kv_state, plan.w_state)
        mz.mz_restore_and_prefill(e, prompt)
        tok, logits = mz.mz_first_token(e, m.vocab)
        report("  first token", restored=tok, clean=clean_tok,
               max_logit_diff=float(np.abs(logits - clean_logits).max()))
        assert float(np.abs(logits - clean_logits).max()) <= LOGIT_TOL
        if tok != clean_tok:
            gap = abs(float(clean_logits[tok] - clean_logits[clean_tok]))
            report("  NEAR-TIE vs clean", gap=gap)
            assert gap <= 2 * LOGIT_TOL
        kv_tol = max(KV_TOL, FLOOR_MARGIN * _floor(key))
        worst_drop = 0.0
        for (l, c), (k0, v0) in pre.items():
            k, v = mz.mz_read_kv(e, l, c, C, dkv)
            state = int(plan.kv_state[l, c])
            if state == W.DROP:
                d = max(float(np.abs(k.astype(np.float64) - k0).max()), float(np.abs(v.astype(np.float64) - v0).max()))
                worst_drop = max(worst_drop, d)
                assert d <= 2 * kv_tol, (key, l, c, state, d)
            else:
                assert k.tobytes() == k0.tobytes(), (key, l, c, state)
                assert v.tobytes() == v0.tobytes(), (key, l, c, state)
        report("  recomputed slots vs clean", max_diff=f"{worst_drop:.3e}")
        got = [mz.mz_read_kv(e, l, 0, C, dkv) for l in range(L)]
        # a context of the first N_ORACLE tokens alone, through every layer
        mz.mz_prefill_context(e, ctx[:N_ORACLE])
        tok64, logits64 = mz.mz_first_token(e, m.vocab)
    finally:
        eng.close()
    Ks, Vs, ologits = _oracle_prefix(m, blob, ctx[:N_ORACLE])
    errs = []
    for l in range(L):
        k, v = got[l]
        errs.append(max(float(np.abs(k[:N_ORACLE].astype(np.float64) - Ks[l]).max()),
                        float(np.abs(v[:N_ORACLE].astype(np.float64) - Vs[l]).max())))
    floor = _floor(key)
    tol = max(KV_TOL, FLOOR_MARGIN * floor)
    worst = max(errs)
    report("  oracle prefix kv", max_err=f"{worst:.3e}", worst_layer=int(np.argmax(errs)),
           layers_within_2e2=int(sum(x <= KV_TOL for x in errs)), half_operand_floor=f"{floor:.3e}",
           tol=f"{tol:.3e}", states_of_chunk0=np.bincount(plan.kv_state[:, 0], minlength=3).tolist())
    assert worst <= tol
    lerr = float(np.abs(logits64.astype(np.float64) - ologits).max())
    otok = O.argmax_first(ologits)
    srt = np.sort(ologits)
    report("  64-token first token", gpu=tok64, oracle=otok, logit_err=f"{lerr:.3e}",
           oracle_margin=f"{float(srt[-1] - srt[-2]):.3e}")
    assert lerr <= LOGIT_TOL
    if tok64 != otok:
        gap = abs(float(ologits[tok64] - ologits[otok]))
        report("  NEAR-TIE", case=key, gap=gap)
        assert gap <= 2 * lerr
