"""Reference eviction planner (TEST INFRASTRUCTURE ONLY, like the rest of
oracle/; shares no code with the library's planner).

What it decides, written from the paper's hybrid-swap policy (Sec. 4.3) and
its backward-out order (Sec. 4.4), re-targeted to two restore paths: the host
link (weights and KV chunks are swapped over it) and GPU recompute (a dropped
KV chunk is rebuilt by the restore's prefill).  The paper hands each increment
of eviction to the path that keeps the two finishing together; here the
recompute path's cost is the restore's FLOP count for the plan, taken from
the row sets the oracle itself uses (restore_rows), because a dropped chunk
drags its rows through every layer up to the one that dropped it.

  order        KV units (layer, chunk) in eviction order:
                 backward-out   layer descending, chunk descending
                 forward-out    layer ascending, chunk ascending
                 token-aligned  chunk descending, then layer descending
                 random-out     backward-out shuffled by Fisher-Yates, the
                                indices drawn from splitmix64(seed)
  weights      n_w units, always swapped: the last layers (the first ones for
               forward-out)
  placement    balanced: a chunk is dropped when the restore's schedule
               finishes earlier with it dropped than with it swapped;
               interleave-2-1: rank r dropped iff r % 3 == 2; all-swap;
               all-drop
  schedule     the link brings the units forward-in, layer by layer, so layer
               l's units have all arrived at A_l = bytes(layers 0..l) / link
               rate; layer l computes after layer l-1 and after A_l:
               end_l = max(end_{l-1}, A_l) + FLOPs_l / recompute rate
               (rates rounded to whole units per second, compared exactly)

Parity is pinned by tests/test_planner.py: it reproduces the stated plans of
the workloads and agrees with the library decision for decision.
"""

from __future__ import annotations

from fractions import Fraction
from typing import List, Tuple

import numpy as np

from .mzoracle import DROP, RES, SWAP, restore_rows

MASK64 = (1 << 64) - 1


def layer_flops(L: int, d: int, dq: int, dkv: int, ff: int, kv_state: np.ndarray, n_ctx: int,
                n_prompt: int, chunk: int) -> List[int]:
    """Per-layer FLOPs of the restore for a plan: queries/attention/MLP for the
    rows carried on (R_{l+1}, or the last position after the last layer) and
    keys/values for the rows written (D_l)."""
    R, D = restore_rows(kv_state, n_ctx, n_prompt, chunk)
    S = n_ctx + n_prompt
    out = []
    for l in range(L):
        q = R[l + 1] if l + 1 < L else np.array([S - 1], dtype=np.int64)
        nq = int(q.size)
        keys = int(np.sum(q + 1))
        out.append(2 * nq * d * 2 * dq + 2 * int(D[l].size) * d * 2 * dkv + 2 * nq * 3 * d * ff + 4 * dq * keys)
    return out


def restore_flops(L: int, d: int, dq: int, dkv: int, ff: int, kv_state: np.ndarray, n_ctx: int,
                  n_prompt: int, chunk: int) -> int:
    return sum(layer_flops(L, d, dq, dkv, ff, kv_state, n_ctx, n_prompt, chunk))


def schedule_end(layer_bytes: List[int], flops: List[int], link_rate: int, recompute_rate: int) -> Fraction:
    """Finish time (s) of the last layer under the forward-in restore schedule."""
    arrive, end = Fraction(0), Fraction(0)
    for b, f in zip(layer_bytes, flops):
        arrive += Fraction(b, link_rate)
        end = max(end, arrive) + Fraction(f, recompute_rate)
    return end


def _splitmix64(state: int) -> Tuple[int, int]:
    state = (state + 0x9E3779B97F4A7C15) & MASK64
    z = state
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return z ^ (z >> 31), state


def eviction_sequence(L: int, nc: int, order: str, seed: int = 0) -> List[Tuple[int, int]]:
    if order == "backward-out" or order == "random-out":
        seq = [(l, c) for l in range(L - 1, -1, -1) for c in range(nc - 1, -1, -1)]
        if order == "random-out":
            x = seed & MASK64
            for i in range(len(seq) - 1, 0, -1):
                r, x = _splitmix64(x)
                j = r % (i + 1)
                seq[i], seq[j] = seq[j], seq[i]
        return seq
    if order == "forward-out":
        return [(l, c) for l in range(L) for c in range(nc)]
    if order == "token-aligned":
        return [(l, c) for c in range(nc - 1, -1, -1) for l in range(L - 1, -1, -1)]
    raise ValueError(order)


def plan_evict(L: int, d: int, dq: int, dkv: int, ff: int, chunk: int, n_ctx: int, n_prompt: int,
               n_kv: int, n_w: int, order: str, placement: str, seed: int, link_rate: float,
               recompute_rate: float, slot_bytes: int, unit_bytes: int, codec: bool = False):
    """(kv_state [L][nc], w_state [L], swapped bytes, restore FLOPs)."""
    nc = (n_ctx + chunk - 1) // chunk
    kv = np.full((L, nc), RES, np.uint8)
    ws = np.full(L, RES, np.uint8)
    link = 0
    layer_bytes = [0] * L
    for i in range(n_w):
        l = i if order == "forward-out" else L - 1 - i
        ws[l] = SWAP
        link += unit_bytes
        layer_bytes[l] += unit_bytes
    bw = int(link_rate + 0.5)
    rf = int(recompute_rate + 0.5)
    seq = eviction_sequence(L, nc, order, seed)
    # a full chunk crosses the link compressed with the codec: n halves take
    # n + n / 16 bytes (oracle/kv_codec.py)
    chunk_bytes = lambda c: (slot_bytes // 2 + slot_bytes // 32
                             if codec and (c + 1) * chunk <= n_ctx else slot_bytes)
    per_layer = lambda plan: layer_flops(L, d, dq, dkv, ff, plan, n_ctx, n_prompt, chunk)
    f_cur = sum(per_layer(kv))
    for r in range(n_kv):
        l, c = seq[r]
        if placement == "all-swap":
            drop = False
        elif placement == "all-drop":
            drop = True
        elif placement == "interleave-2-1":
            drop = r % 3 == 2
        elif placement == "balanced":
            with_swap = list(layer_bytes)
            with_swap[l] += chunk_bytes(c)
            if_swap = schedule_end(with_swap, per_layer(kv), bw, rf)
            trial = kv.copy()
            trial[l, c] = DROP
            if_drop = schedule_end(layer_bytes, per_layer(trial), bw, rf)
            drop = if_drop < if_swap
        else:
            raise ValueError(placement)
        if drop:
            kv[l, c] = DROP
            f_cur = sum(per_layer(kv))
        else:
            kv[l, c] = SWAP
            link += chunk_bytes(c)
            layer_bytes[l] += chunk_bytes(c)
    return kv, ws, link, f_cur
