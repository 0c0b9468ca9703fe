"""Rounding floor of reduced-precision GEMM operands over the depth of the model.

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
a token prefix twice, once in fp64 and once with operand roundings, and
reports how far apart the stored (half) keys and values end up at each layer.
Keys and values are stored as half in both runs, as the KV cache is.

Which operands are rounded, and to what, is a Rounding: weights (the
dequantized matrices), activations (every other product input), and the
attention probabilities that multiply V, each "exact", "half" or "bf16"
(round to nearest even).  The half-operand floor is weights and activations
in half, probabilities exact.

Parity unpinned beyond its special cases: with every rounding switched off it
reproduces the fp64 oracle's keys and values bit for bit, and with weights
and activations in half it equals the half-operand floor (both pinned in
tests/test_oracle_pins.py); the size of a floor is a measurement, not a
closed form.
"""

from __future__ import annotations

import math
from typing import Callable, List, NamedTuple, Tuple

import numpy as np

from .mzoracle import Hyper, Weights, causal_gqa_attention, rmsnorm, rope, silu


def _half(a: np.ndarray) -> np.ndarray:
    return np.asarray(a, dtype=np.float64).astype(np.float16).astype(np.float64)


def _bf16(a: np.ndarray) -> np.ndarray:
    """Round to the nearest bfloat16 (8 significant bits), ties to even, via
    the top 16 bits of the float32 that holds the value after rounding."""
    x = np.asarray(a, dtype=np.float64).astype(np.float32)
    b = x.view(np.uint32).astype(np.uint64)
    b = (b + 0x7FFF + ((b >> 16) & 1)) & 0xFFFF0000
    return b.astype(np.uint32).view(np.float32).astype(np.float64)


def _ident(a: np.ndarray) -> np.ndarray:
    return a


ROUND = {"exact": _ident, "half": _half, "bf16": _bf16}


class Rounding(NamedTuple):
    weights: str = "exact"
    acts: str = "exact"
    probs: str = "exact"


HALF_OPERANDS = Rounding("half", "half", "exact")
EXACT = Rounding()


def _attention_rounded_probs(q, pos, K, V, rp):
    """causal_gqa_attention with the softmax probabilities rounded by rp
    before they multiply V (queries one at a time; for short prefixes)."""
    n, nq, hd = q.shape
    nkv = K.shape[1]
    group = nq // nkv
    out = np.empty_like(q)
    for i in range(n):
        last = int(pos[i]) + 1
        for h in range(nq):
            g = h // group
            s = K[:last, g] @ q[i, h] / math.sqrt(hd)
            p = np.exp(s - s.max())
            p = rp(p / p.sum())
            out[i, h] = p @ V[:last, g]
    return out


def prefix_kv(hp: Hyper, wts: Weights, tokens: np.ndarray, rounding,
              progress: Callable[[int], None] = None) -> Tuple[List[np.ndarray], List[np.ndarray], np.ndarray]:
    """Keys and values (float64 of the stored half values, [L][n, dkv]) of a
    prefill over `tokens`, and the final hidden state of the last row, with
    the operands rounded as `rounding` says (True: the half-operand floor's
    rounding; False: none)."""
    if rounding is True:
        rounding = HALF_OPERANDS
    elif rounding is False:
        rounding = EXACT
    rw, ra, rp = ROUND[rounding.weights], ROUND[rounding.acts], ROUND[rounding.probs]
    tokens = np.asarray(tokens, dtype=np.int64)
    n = tokens.size
    pos = np.arange(n)
    h = wts.rows("emb", tokens)
    Ks, Vs = [], []
    for l in range(hp.n_layers):
        w = wts.layer(l)
        wq, wk, wv, wo, wg, wu, wd = (rw(w[k]) for k in ("wq", "wk", "wv", "wo", "wg", "wu", "wd"))
        x = ra(rmsnorm(h, hp.rms_eps))
        q = rope((x @ wq.T).reshape(n, hp.n_q_heads, hp.head_dim), pos, hp.rope_theta)
        k = rope((x @ wk.T).reshape(n, hp.n_kv_heads, hp.head_dim), pos, hp.rope_theta)
        v = (x @ wv.T).reshape(n, hp.n_kv_heads, hp.head_dim)
        K = _half(k.reshape(n, hp.dkv))
        V = _half(v.reshape(n, hp.dkv))
        Ks.append(K)
        Vs.append(V)
        Kh = K.reshape(n, hp.n_kv_heads, hp.head_dim)
        Vh = V.reshape(n, hp.n_kv_heads, hp.head_dim)
        if rounding.probs == "exact":
            o = causal_gqa_attention(ra(q), pos, Kh, Vh)
        else:
            o = _attention_rounded_probs(ra(q), pos, Kh, Vh, rp)
        h = h + ra(o.reshape(n, hp.dq)) @ wo.T
        y = ra(rmsnorm(h, hp.rms_eps))
        h = h + ra(silu(y @ wg.T) * (y @ wu.T)) @ wd.T
        if progress:
            progress(l)
    return Ks, Vs, h[-1]


def kv_distance(A: Tuple[List[np.ndarray], List[np.ndarray]], B) -> np.ndarray:
    """Per layer: max |K, V of A - K, V of B|."""
    return np.array([max(np.abs(a - b).max(), np.abs(c - d).max())
                     for a, b, c, d in zip(A[0], B[0], A[1], B[1])])


def f16_operand_floor(hp: Hyper, wts: Weights, tokens: np.ndarray,
                      progress: Callable[[str, int], None] = None) -> np.ndarray:
    """Per layer: max |K, V (half operands) - K, V (fp64)| over the prefix."""
    K0, V0, _ = prefix_kv(hp, wts, tokens, False, progress and (lambda l: progress("fp64", l)))
    K1, V1, _ = prefix_kv(hp, wts, tokens, True, progress and (lambda l: progress("half", l)))
    return kv_distance((K1, V1), (K0, V0))
