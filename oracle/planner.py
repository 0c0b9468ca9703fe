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
                                indices drawn from splitmix64(seed) (Steele,
                                Lea and Flood, OOPSLA 2014)
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

import math
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


# --------------------------------------------------------------------------
# Size-driven eviction: the hybrid-swap policy (Sec. 4.3, Alg. 1), taken one
# unit at a time in backward-out order (Sec. 4.4) until the requested bytes
# are released (the evict(size) interface of Sec. 5).
#
# Paths: the link (weight layers, swapped chunks) plays the storage path of
# the paper, the one weights are tied to; recompute (dropped chunks) plays
# the in-memory decompression path, which takes KV chunks only.  Stages, from
# the counts N_KV / N_W of resident evictable units (Alg. 1):
#   N_KV > T              KV_ONLY   chunk to the path that stays behind
#   N_KV > 0 and N_W > 0  KV_AND_W  weight layers, each followed by the KV
#                                   chunks its reload covers, all dropped
#                                   (paper rule: also while the last weight
#                                   layer taken still covers chunks)
#   N_KV > 0, N_W = 0               the KV_ONLY rule (no weight left)
#   N_W > 0               W_ONLY    a weight layer
#   else                  EXHAUSTED (the paper's CompKV has no counterpart:
#                                    nothing compressed stays on the device)
#
# Two rules for T and the KV_AND_W pairing:
#   "paper" (default)  the paper's: with per-unit times t_d (one KV chunk on
#                      the recompute path) and t_W (one weight layer over the
#                      link), k = floor(t_W / t_d) chunks are dropped per
#                      weight layer and T = N_W^total * k.  A chunk's
#                      recompute time is not a constant on this engine; t_d
#                      is the per-unit time of the front-most chunk (chunk 0
#                      of layer 0, the unit restored last in backward-out
#                      order) dropped alone: its rows' layer-0 K/V projection.
#   "total"            every time a path total over the plan: T = the largest
#                      n for which dropping the n front-most chunks costs no
#                      more recompute than reloading all N_W^total weight
#                      layers; in KV_AND_W a chunk is dropped while the
#                      recompute total with it stays within the link total,
#                      else the next weight layer goes.  With a constant t_d
#                      this T is floor(N_W^total * t_W / t_d), which carries
#                      the fractions of one layer's share into the next.
# In KV_ONLY (both rules) the chunk goes to recompute iff the recompute total
# with it stays below the link total with it swapped (the split in inverse
# proportion to the two per-unit times, with the plan's exact costs).

KV_ONLY, KV_AND_W, W_ONLY, EXHAUSTED = 0, 1, 2, 3


def paper_threshold(n_w_total, t_w, t_d):
    """(T, k): k = floor(t_W / t_d) chunks per weight layer, T = N_W^total * k
    (Sec. 4.3)."""
    k = math.floor(Fraction(t_w) / Fraction(t_d)) if t_d > 0 else 0
    return n_w_total * k, k


def total_threshold(kv_seq, rec_time, n_w_total, t_w):
    """T of the "total" rule: front-most chunks (the tail of kv_seq) whose
    recompute fits the reload of all evictable weight layers."""
    T = 0
    budget = n_w_total * t_w
    for n in range(1, len(kv_seq) + 1):
        if rec_time(set(kv_seq[len(kv_seq) - n:])) > budget:
            break
        T = n
    return T


def hybrid_swap_evict(kv_seq, w_seq, kv_state, w_state, T, request, kv_release, w_release, kv_link, w_link,
                      rec_time, k=None):
    """One evict(size) call.

    kv_seq / w_seq: every evictable chunk / weight id in eviction order;
    kv_state / w_state: dicts id -> RES / SWAP / DROP, updated in place;
    kv_link(id), w_link: link time of a unit; rec_time(set of dropped chunk
    ids): recompute time of that plan's extra work.  k: chunks per weight
    layer in KV_AND_W (the paper's rule); None for the "total" rule.  Returns
    (evicted ids with their stage, released bytes)."""
    dropped = {u for u, s in kv_state.items() if s == DROP}
    link = sum((kv_link(u) for u, s in kv_state.items() if s == SWAP), Fraction(0))
    link += sum((w_link for s in w_state.values() if s != RES), Fraction(0))
    taken, released = [], 0

    def counts():
        return (sum(1 for u in kv_seq if kv_state[u] == RES), sum(1 for u in w_seq if w_state[u] == RES))

    def owed(n_kv, n_w):
        # paper rule: the weight layers taken in KV_AND_W still cover chunks
        # not yet taken (the stage began at N_KV = min(T, all chunks))
        return k is not None and min(T, len(kv_seq)) - n_kv < k * (len(w_seq) - n_w)

    def stage():
        n_kv, n_w = counts()
        if n_kv > T:
            return KV_ONLY
        if n_kv > 0 and (n_w > 0 or owed(n_kv, n_w)):
            return KV_AND_W
        if n_kv > 0:
            return KV_ONLY
        return W_ONLY if n_w > 0 else EXHAUSTED

    def evict_weight(st):
        nonlocal link, released
        u = next(u for u in w_seq if w_state[u] == RES)
        w_state[u] = DROP
        link += w_link
        released += w_release
        taken.append((("w", u), st))

    while released < request:
        st = stage()
        if st == EXHAUSTED:
            break
        if st == W_ONLY:
            evict_weight(st)
            continue
        if st == KV_AND_W and k is not None:
            # a weight layer, then the k chunks its reload covers
            n_kv, n_w = counts()
            if n_w > 0 and not owed(n_kv, n_w):
                evict_weight(st)
                continue
        u = next(u for u in kv_seq if kv_state[u] == RES)
        rec_with = rec_time(dropped | {u})
        if st == KV_AND_W and k is None and rec_with > link:
            evict_weight(st)
            continue
        if st == KV_AND_W or rec_with < link + kv_link(u):
            kv_state[u] = DROP
            dropped.add(u)
        else:
            kv_state[u] = SWAP
            link += kv_link(u)
        released += kv_release
        taken.append((("kv", u), st))
    return taken, released


def plan_evict_size(L: int, d: int, dq: int, dkv: int, ff: int, chunk: int, n_ctx: int, n_prompt: int,
                    kv_state: np.ndarray, w_state: np.ndarray, request: int, n_w_total: int, link_rate: float,
                    recompute_rate: float, slot_bytes: int, unit_bytes: int, codec: bool = False,
                    rule: str = "paper"):
    """The policy on this engine's restore: chunk (l, c) and weight layer l,
    link times from bytes, recompute time from the restore's FLOP count.
    Returns (kv_state, w_state, unit ids in order with stages, released, T)."""
    nc = (n_ctx + chunk - 1) // chunk
    bw = int(link_rate + 0.5)
    rf = int(recompute_rate + 0.5)
    kv_seq = [(l, c) for l in range(L - 1, -1, -1) for c in range(nc - 1, -1, -1)]
    w_seq = list(range(L - 1, L - 1 - n_w_total, -1))

    def flops_of(dropped):
        plan = np.full((L, nc), RES, np.uint8)
        for l, c in dropped:
            plan[l, c] = DROP
        return restore_flops(L, d, dq, dkv, ff, plan, n_ctx, n_prompt, chunk)

    f0 = flops_of(set())
    rec_time = lambda dropped: Fraction(flops_of(dropped) - f0, rf)
    kv_link = lambda u: Fraction(slot_bytes // 2 + slot_bytes // 32
                                 if codec and (u[1] + 1) * chunk <= n_ctx else slot_bytes, bw)
    w_link = Fraction(unit_bytes, bw)
    if rule == "paper":
        T, k = paper_threshold(n_w_total, w_link, rec_time({(0, 0)}))
    elif rule == "total":
        T, k = total_threshold(kv_seq, rec_time, n_w_total, w_link), None
    else:
        raise ValueError(rule)
    kvs = {(l, c): int(kv_state[l, c]) for l in range(L) for c in range(nc)}
    ws = {l: int(w_state[l]) for l in range(L)}
    taken, released = hybrid_swap_evict(kv_seq, w_seq, kvs, ws, T, request, slot_bytes, unit_bytes, kv_link,
                                        w_link, rec_time, k)
    out_kv = np.array([[kvs[(l, c)] for c in range(nc)] for l in range(L)], np.uint8)
    out_w = np.array([ws[l] for l in range(L)], np.uint8)
    ids = [u[0] * nc + u[1] if kind == "kv" else L * nc + u for (kind, u), _ in taken]
    stages = [st for _, st in taken]
    return out_kv, out_w, ids, stages, released, T
