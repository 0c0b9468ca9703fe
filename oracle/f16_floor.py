"""Rounding floor of half-precision GEMM operands over the depth of the model.

TEST INFRASTRUCTURE ONLY (like the rest of oracle/): it sets a tolerance, it is
never called by the product path, and it shares no code with it.

The fp64 oracle (mzoracle) is the parity reference.  An implementation that
feeds its matrix products with IEEE half operands -- dequantized weights
d * (q - 8) rounded to half, and half activations at every product input (the
RMSNorm outputs, the rotated queries, the attention output, the SwiGLU
output), with exact accumulation -- cannot stay closer to that reference than
the rounding itself allows, and after many layers the rounding of one layer
has moved every later layer's input.  This module runs the oracle's layer
(paper Sec. 2.1: the prefill that produces each layer's keys and values) over
a token prefix twice, once in fp64 and once with those half-precision operand
roundings, and reports how far apart the stored (half) keys and values end up
at each layer.  Keys and values are stored as half in both runs, as the
KV cache is.

Parity unpinned beyond its special case: with every rounding switched off it
reproduces the fp64 oracle's keys and values bit for bit (pinned in
tests/test_oracle_pins.py); the size of the floor is a measurement, not a
closed form.
"""

from __future__ import annotations

from typing import Callable, List, Tuple

import numpy as np

from .mzoracle import Hyper, Weights, causal_gqa_attention, rmsnorm, rope, silu


def _half(a: np.ndarray) -> np.ndarray:
    return np.asarray(a, dtype=np.float64).astype(np.float16).astype(np.float64)


def _ident(a: np.ndarray) -> np.ndarray:
    return a


def prefix_kv(hp: Hyper, wts: Weights, tokens: np.ndarray, half_operands: bool,
              progress: Callable[[int], None] = None) -> Tuple[List[np.ndarray], List[np.ndarray], np.ndarray]:
    """Keys and values (float64 of the stored half values, [L][n, dkv]) of a
    prefill over `tokens`, and the final hidden state of the last row.  With
    half_operands, every matrix-product operand is rounded to half first."""
    r = _half if half_operands else _ident
    tokens = np.asarray(tokens, dtype=np.int64)
    n = tokens.size
    pos = np.arange(n)
    h = wts.rows("emb", tokens)
    Ks, Vs = [], []
    for l in range(hp.n_layers):
        w = wts.layer(l)
        wq, wk, wv, wo, wg, wu, wd = (r(w[k]) for k in ("wq", "wk", "wv", "wo", "wg", "wu", "wd"))
        x = r(rmsnorm(h, hp.rms_eps))
        q = rope((x @ wq.T).reshape(n, hp.n_q_heads, hp.head_dim), pos, hp.rope_theta)
        k = rope((x @ wk.T).reshape(n, hp.n_kv_heads, hp.head_dim), pos, hp.rope_theta)
        v = (x @ wv.T).reshape(n, hp.n_kv_heads, hp.head_dim)
        K = _half(k.reshape(n, hp.dkv))
        V = _half(v.reshape(n, hp.dkv))
        Ks.append(K)
        Vs.append(V)
        o = causal_gqa_attention(r(q), pos, K.reshape(n, hp.n_kv_heads, hp.head_dim),
                                 V.reshape(n, hp.n_kv_heads, hp.head_dim))
        h = h + r(o.reshape(n, hp.dq)) @ wo.T
        y = r(rmsnorm(h, hp.rms_eps))
        h = h + r(silu(y @ wg.T) * (y @ wu.T)) @ wd.T
        if progress:
            progress(l)
    return Ks, Vs, h[-1]


def f16_operand_floor(hp: Hyper, wts: Weights, tokens: np.ndarray,
                      progress: Callable[[str, int], None] = None) -> np.ndarray:
    """Per layer: max |K, V (half operands) - K, V (fp64)| over the prefix."""
    K0, V0, _ = prefix_kv(hp, wts, tokens, False, progress and (lambda l: progress("fp64", l)))
    K1, V1, _ = prefix_kv(hp, wts, tokens, True, progress and (lambda l: progress("half", l)))
    return np.array([max(np.abs(a - b).max(), np.abs(c - d).max()) for a, b, c, d in zip(K1, K0, V1, V0)])
