"""Size-driven eviction (mz_plan_evict_size): the hybrid-swap state machine
(Sec. 4.3, Alg. 1) pinned on its closed forms, and the library's planner
against the reference in oracle/ decision for decision.  CPU only."""

import math
from fractions import Fraction

import numpy as np
import pytest

import oracle as O
from oracle.planner import (EXHAUSTED, KV_AND_W, KV_ONLY, W_ONLY, hybrid_swap_evict, paper_threshold,
                            plan_evict_size, restore_flops, total_threshold)
from paper_2609_01338_amd import mz
from paper_2609_01338_amd import workloads as W

# ---------------------------------------------------------------------------
# the state machine with constant per-unit times: the paper's own model


def _const_machine(n_kv, n_w_total, t_l, t_d, t_w, rule="paper"):
    kv_seq = list(range(n_kv))
    w_seq = list(range(n_w_total))
    rec = lambda s: len(s) * t_d
    if rule == "paper":
        T, k = paper_threshold(n_w_total, t_w, t_d)
    else:
        T, k = total_threshold(kv_seq, rec, n_w_total, t_w), None
    kvs = {u: O.RES for u in kv_seq}
    ws = {u: O.RES for u in range(n_w_total)}
    return kv_seq, w_seq, rec, T, k, kvs, ws


def _run(kv_seq, w_seq, kvs, ws, T, k, request, t_l, t_w, rec):
    return hybrid_swap_evict(kv_seq, w_seq, kvs, ws, T, request, 1, 1, lambda u: t_l, t_w, rec, k)


CONST = [  # n_kv, n_w_total, t_l, t_d, t_w
    (200, 8, Fraction(1), Fraction(3), Fraction(10)),
    (200, 8, Fraction(5), Fraction(2), Fraction(7)),
    (50, 10, Fraction(1), Fraction(1), Fraction(9)),       # n_kv <= T: starts in KV_AND_W
    (300, 4, Fraction(2, 3), Fraction(7, 5), Fraction(17, 2)),
    (120, 0, Fraction(1), Fraction(2), Fraction(5)),       # no evictable weights: T = 0
    (100, 6, Fraction(1), Fraction(4), Fraction(3)),       # t_W < t_d: k = 0, T = 0
]


def test_threshold_paper_formula():
    """Sec. 4.3: while one weight layer reloads, the other path restores
    floor(t_W / t_d) chunks, so T = N_W^total * floor(t_W / t_d); e.g. eight
    layers with t_W = 7 and t_d = 2 give 8 * 3 = 24 (not floor(56 / 2) = 28)."""
    assert paper_threshold(8, Fraction(7), Fraction(2)) == (24, 3)
    assert paper_threshold(0, Fraction(7), Fraction(2)) == (0, 3)
    assert paper_threshold(5, Fraction(1), Fraction(2)) == (0, 0)


@pytest.mark.parametrize("n_kv,n_w,t_l,t_d,t_w", CONST)
def test_threshold_closed_form(n_kv, n_w, t_l, t_d, t_w):
    """Paper rule: T = N_W^total floor(t_W / t_d), whatever the number of
    chunks.  Total rule: the front-most chunks whose recompute fits the whole
    reload, floor(N_W^total t_W / t_d) capped by the number of chunks."""
    *_, T, k, _, _ = _const_machine(n_kv, n_w, t_l, t_d, t_w)
    assert k == math.floor(t_w / t_d) and T == n_w * math.floor(t_w / t_d)
    *_, T, k, _, _ = _const_machine(n_kv, n_w, t_l, t_d, t_w, "total")
    assert k is None and T == min(n_kv, math.floor(n_w * t_w / t_d))


@pytest.mark.parametrize("n_kv,n_w,t_l,t_d,t_w", CONST)
def test_stage_sequence_and_split(n_kv, n_w, t_l, t_d, t_w):
    kv_seq, w_seq, rec, T, k, kvs, ws = _const_machine(n_kv, n_w, t_l, t_d, t_w)
    taken, released = _run(kv_seq, w_seq, kvs, ws, T, k, 10 ** 9, t_l, t_w, rec)
    stages = [st for _, st in taken]
    kinds = [kind for (kind, _), _ in taken]
    # everything evictable is taken, each unit once
    assert released == n_kv + n_w and len(taken) == n_kv + n_w
    assert all(kvs[u] != O.RES for u in kv_seq) and all(ws[u] != O.RES for u in w_seq)
    # weights leave only as the rearmost first
    assert [u for (kind, u), _ in taken if kind == "w"] == w_seq
    # KV_ONLY while more than T chunks remain, weights untouched
    n_kv_only = max(0, n_kv - T)
    assert stages[:n_kv_only] == [KV_ONLY] * n_kv_only
    assert all(kind == "kv" for kind in kinds[:n_kv_only])
    # KV_ONLY split in inverse proportion to the unit times: the two totals
    # stay within one unit of each other
    drops = sum(1 for (kind, u), _ in taken[:n_kv_only] if kvs[u] == O.DROP)
    swaps = n_kv_only - drops
    assert abs(drops * t_d - swaps * t_l) <= max(t_l, t_d)
    if n_kv_only:
        assert abs(drops - n_kv_only * t_l / (t_l + t_d)) <= 1
    # KV_AND_W: each weight layer followed by exactly k dropped chunks
    rest = taken[n_kv_only:]
    pair = [(kind, st) for (kind, _), st in rest if st == KV_AND_W]
    if n_w and min(n_kv, T) > 0:
        groups = min(n_w, -(-min(n_kv, T) // k))
        expect = []
        left = min(n_kv, T)
        for _ in range(groups):
            expect += [("w", KV_AND_W)] + [("kv", KV_AND_W)] * min(k, left)
            left -= min(k, left)
        assert pair == expect
        assert all(kvs[u] == O.DROP for (kind, u), st in rest if kind == "kv" and st == KV_AND_W)
    if n_kv > T and n_w and k:
        # N_KV equals T at the transition: chunks and weight layers run out together
        assert rest == [r for r in rest if r[1] == KV_AND_W] and len(rest) == n_w * (k + 1)
    if n_kv <= T and n_w:
        # the chunks run out first; the rest are weights alone
        assert stages[0] == KV_AND_W
        last_kv = max(i for i, kind in enumerate(kinds) if kind == "kv")
        assert all(st == W_ONLY for _, st in taken[last_kv + 1:])
    if T == 0:
        assert set(stages) <= {KV_ONLY, W_ONLY} and stages[:n_kv] == [KV_ONLY] * n_kv


@pytest.mark.parametrize("n_kv,n_w,t_l,t_d,t_w", CONST[:4])
def test_balance_preserved_wherever_eviction_stops(n_kv, n_w, t_l, t_d, t_w):
    """Through KV_ONLY the two path totals stay within one chunk of each
    other.  Through KV_AND_W each increment is a weight layer and the k
    chunks its reload covers: it adds t_W to the link and k t_d to
    recompute, which differ by less than one chunk (t_W - k t_d in [0, t_d)),
    so any stopping point is balanced to that grain plus one weight layer."""
    kv_seq, w_seq, rec, T, k, kvs, ws = _const_machine(n_kv, n_w, t_l, t_d, t_w)
    link = Fraction(0)
    rec_t = Fraction(0)
    m = max(t_l, t_d)
    at_entry = None
    groups = 0
    while True:
        taken, _ = _run(kv_seq, w_seq, kvs, ws, T, k, 1, t_l, t_w, rec)
        if not taken:
            break
        (kind, u), st = taken[0]
        if kind == "w":
            link += t_w
        elif kvs[u] == O.SWAP:
            link += t_l
        else:
            rec_t += t_d
        if st == KV_ONLY and sum(1 for v in kv_seq if kvs[v] == O.RES) > T:
            assert abs(link - rec_t) <= m
        if st == KV_AND_W:
            if at_entry is None:
                at_entry = (link - t_w) - rec_t if kind == "w" else link - (rec_t - t_d)
            groups += kind == "w"
            assert 0 <= t_w - k * t_d < t_d
            assert abs(link - rec_t) <= abs(at_entry) + t_w + groups * (t_w - k * t_d)


def test_total_rule_pairs_by_path_totals():
    """The "total" rule keeps the two totals level through KV_AND_W (a
    weight layer goes once recompute would pass the link)."""
    kv_seq, w_seq, rec, T, k, kvs, ws = _const_machine(200, 8, Fraction(5), Fraction(2), Fraction(7), "total")
    taken, _ = _run(kv_seq, w_seq, kvs, ws, T, k, 10 ** 9, Fraction(5), Fraction(7), rec)
    assert T == 28
    link = rec_t = Fraction(0)
    for (kind, u), st in taken:
        if kind == "w":
            link += 7
        elif kvs[u] == O.SWAP:
            link += 5
        else:
            rec_t += 2
        if st == KV_AND_W:
            assert rec_t <= link + 7


@pytest.mark.parametrize("rule", ["paper", "total"])
def test_calls_continue_where_the_last_stopped(rule):
    """A sequence of calls takes exactly the units of one call for their
    total: the state machine keeps no state beside the units' states."""
    args = (200, 8, Fraction(1), Fraction(3), Fraction(10))
    kv_seq, w_seq, rec, T, k, kvs, ws = _const_machine(*args, rule)
    full, _ = _run(kv_seq, w_seq, kvs, ws, T, k, 10 ** 9, args[2], args[4], rec)
    kv_seq, w_seq, rec, T, k, kvs, ws = _const_machine(*args, rule)
    got = []
    for req in (3, 1, 17, 60, 2, 10 ** 9):
        t, r = _run(kv_seq, w_seq, kvs, ws, T, k, req, args[2], args[4], rec)
        assert r >= min(req, len(full) - len(got))
        got += t
    assert got == full
    t, r = _run(kv_seq, w_seq, kvs, ws, T, k, 5, args[2], args[4], rec)
    assert t == [] and r == 0                                           # exhausted


# ---------------------------------------------------------------------------
# the work model that prices a dropped chunk


def test_front_chunk_costs_its_layer0_kv_projection():
    """Dropping a chunk of layer 0 alone adds exactly its rows' K/V
    projection at layer 0: 2 rows d 2dkv FLOPs (R_1 and every later set are
    unchanged, so nothing else is recomputed)."""
    L, d, dq, dkv, ff, C, N = 4, 256, 256, 128, 512, 64, 200
    base = np.zeros((L, (N + C - 1) // C), np.uint8)
    f0 = restore_flops(L, d, dq, dkv, ff, base, N, 0, C)
    for c, rows in [(0, 64), (3, N - 3 * C)]:
        p = base.copy()
        p[0, c] = O.DROP
        assert restore_flops(L, d, dq, dkv, ff, p, N, 0, C) - f0 == 2 * rows * d * 2 * dkv


# ---------------------------------------------------------------------------
# library planner vs the reference, decision for decision


def _setup(shape):
    L, d, nq, nkv, hd, ff, C, n_ctx, n_prompt = shape
    m = W.ModelConfig("t", L, d, nq, nkv, hd, ff, 1024, 1e4, C)
    cfg = mz.make_cfg(m, n_ctx + n_prompt)
    _, _, e = mz.mz_plan_evict(cfg, n_ctx, 0, 0, 1, "backward-out", "all-swap")
    unit = int(e["swap_bytes"])
    slot = C * nkv * hd * 4
    return m, cfg, unit, slot


SHAPES = [
    # L, d, nq, nkv, hd, ff, C, n_ctx, n_prompt
    (3, 256, 4, 2, 64, 688, 64, 700, 0),
    (4, 512, 8, 2, 64, 1024, 128, 1024, 16),
    (5, 256, 4, 4, 64, 512, 64, 448, 5),
]
RATES = [(1e7, 1e10), (1e8, 1e9), (3e6, 1e11), (5.5e7, 2.5e10)]


@pytest.mark.parametrize("rule", ["paper", "total"])
@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("rates", RATES)
def test_matches_reference_over_calls(shape, rates, rule):
    L, d, nq, nkv, hd, ff, C, n_ctx, n_prompt = shape
    m, cfg, unit, slot = _setup(shape)
    nc = (n_ctx + C - 1) // C
    link, rec = rates
    rng = np.random.default_rng(hash((shape, rates, rule)) % 2 ** 32)
    for trial in range(2):
        codec = trial == 1
        n_w_total = int(rng.integers(0, L + 1))
        kv = np.zeros((L, nc), np.uint8)
        ws = np.zeros(L, np.uint8)
        okv, ows = kv.copy(), ws.copy()
        total = 0
        while True:
            req = int(rng.integers(1, 6)) * slot + int(rng.integers(0, 2)) * unit
            kv, ws, order, stage, info = mz.mz_plan_evict_size(cfg, n_ctx, kv, ws, req, link, rec, n_w_total,
                                                                n_prompt, codec, rule)
            okv, ows, oids, ost, orel, oT = plan_evict_size(L, d, nq * hd, nkv * hd, ff, C, n_ctx, n_prompt, okv,
                                                            ows, req, n_w_total, link, rec, slot, unit, codec, rule)
            assert np.array_equal(kv, okv) and np.array_equal(ws, ows)
            assert list(order) == oids and list(stage) == ost
            assert info["released"] == orel and info["T"] == oT
            assert info["reached"] == (orel >= req)
            total += orel
            if not info["reached"]:
                assert info["stage"] == "exhausted" and info["n_kv"] == 0 and info["n_w"] == 0
                break
        # everything evictable is gone; weights beyond n_w_total never move
        assert not (kv == O.RES).any()
        assert list(ws) == [O.RES] * (L - n_w_total) + [O.DROP] * n_w_total
        assert total == L * nc * slot + n_w_total * unit


@pytest.mark.parametrize("rule", ["paper", "total"])
def test_matches_reference_from_a_mixed_state(rule):
    """Starting from a state left by an explicit plan (swapped and dropped
    chunks, a swapped weight layer) the totals include what is already out."""
    shape = (4, 512, 8, 2, 64, 1024, 128, 1024, 16)
    L, d, nq, nkv, hd, ff, C, n_ctx, n_prompt = shape
    m, cfg, unit, slot = _setup(shape)
    p = W.random_plan(L, (n_ctx + C - 1) // C, 0.3, 0.2, 4, w_swap=0.3, w_drop=0.0)
    for req in (slot, 7 * slot, 10 ** 12):
        a = mz.mz_plan_evict_size(cfg, n_ctx, p.kv_state, p.w_state, req, 2e7, 3e10, L, n_prompt, rule=rule)
        b = plan_evict_size(L, d, nq * hd, nkv * hd, ff, C, n_ctx, n_prompt, p.kv_state, p.w_state, req, L,
                            2e7, 3e10, slot, unit, rule=rule)
        assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1]) and list(a[2]) == b[2]
        assert list(a[3]) == b[3] and a[4]["released"] == b[4]


def test_workload_8b_stages():
    """On the 8B context.  Paper rule: t_d is chunk 0 of layer 0's K/V
    projection (2 * 256 * 4096 * 2048 FLOPs), so floor(t_W / t_d) of them fit
    one weight reload and T = 32 of those exceeds the 4096 chunks: eviction
    starts in KV_AND_W (the paper's second case), a weight layer then its k
    chunks, until the chunks run out.  Total rule: the front-most chunks that
    the weight reload covers are a few of the 4096, so it starts in KV_ONLY
    and reaches KV_AND_W before the context is gone."""
    w = W.WORKLOADS["8b"]
    m = w.model
    cfg = mz.make_cfg(m, w.n_ctx + w.n_prompt)
    L, nc = m.n_layers, w.n_chunks
    kv = np.zeros((L, nc), np.uint8)
    ws = np.zeros(L, np.uint8)
    slot = m.chunk_tokens * m.dkv * 4
    _, _, e = mz.mz_plan_evict(cfg, w.n_ctx, 0, 0, 1, "backward-out", "all-swap")
    unit = int(e["swap_bytes"])
    link, rec = 56e9, 4e14
    k = math.floor(Fraction(unit, int(link)) / Fraction(2 * 256 * m.d_model * 2 * m.dkv, int(rec)))
    kv2, ws2, order, stage, info = mz.mz_plan_evict_size(cfg, w.n_ctx, kv, ws, 10 ** 13, link, rec, L,
                                                         w.n_prompt, True)
    assert info["T"] == L * k and L * k > L * nc
    assert stage[0] == KV_AND_W and order[0] == L * nc + L - 1            # weight layer 31 first
    assert list(order[1:k + 1]) == list(range(L * nc - 1, L * nc - 1 - k, -1))   # then k chunks, rearmost first
    assert info["stage"] == "exhausted" and not info["reached"]
    kv3, ws3, order3, _, info3 = mz.mz_plan_evict_size(cfg, w.n_ctx, kv, ws, 100 * slot, link, rec, L,
                                                       w.n_prompt, True)
    assert list(order3) == list(order[:len(order3)]) and info3["released"] >= 100 * slot
    # the total rule
    kv2, ws2, order, stage, info = mz.mz_plan_evict_size(cfg, w.n_ctx, kv, ws, 10 ** 13, link, rec, L,
                                                         w.n_prompt, True, "total")
    assert 0 < info["T"] < L * nc
    assert stage[0] == KV_ONLY and KV_AND_W in set(stage.tolist())
    assert info["stage"] == "exhausted" and not info["reached"]
    kv3, ws3, order3, _, info3 = mz.mz_plan_evict_size(cfg, w.n_ctx, kv, ws, 100 * slot, link, rec, L,
                                                       w.n_prompt, True, "total")
    assert list(order3) == list(order[:100]) and info3["released"] == 100 * slot


def test_errors():
    w = W.WORKLOADS["tiny"]
    cfg = mz.make_cfg(w.model, w.n_ctx)
    L, nc = w.model.n_layers, w.n_chunks
    kv = np.zeros((L, nc), np.uint8)
    ws = np.zeros(L, np.uint8)
    with pytest.raises(mz.MzError):
        mz.mz_plan_evict_size(cfg, w.n_ctx, kv, ws, 100, 0.0, 1e9, L)           # no link rate
    with pytest.raises(mz.MzError):
        mz.mz_plan_evict_size(cfg, w.n_ctx, kv, ws, 100, 1e9, 1e9, L + 1)       # n_w_total
    with pytest.raises(mz.MzError):
        mz.mz_plan_evict_size(cfg, w.n_ctx, kv, ws, -1, 1e9, 1e9, L)            # bytes
    bad = kv.copy()
    bad[0, 0] = 7
    with pytest.raises(mz.MzError):
        mz.mz_plan_evict_size(cfg, w.n_ctx, bad, ws, 100, 1e9, 1e9, L)
    # nothing requested: nothing taken
    kv2, ws2, order, _, info = mz.mz_plan_evict_size(cfg, w.n_ctx, kv, ws, 0, 1e9, 1e9, L)
    assert order.size == 0 and info["released"] == 0 and info["reached"]
    with pytest.raises(KeyError):
        mz.mz_plan_evict_size(cfg, w.n_ctx, kv, ws, 100, 1e9, 1e9, L, rule="other")
    req = mz.mz_evict_size_request(100, 0, L, 1e9, 1e9, 0, 7)            # unknown rule value
    info = np.zeros(8)
    n = mz.ctypes.c_int32()
    o = np.empty(L * (nc + 1), np.int32)
    st = mz.lib().mz_plan_evict_size(mz.ctypes.byref(cfg), w.n_ctx, mz.ctypes.byref(req), kv.ctypes.data,
                                     ws.ctypes.data, o.ctypes.data, None, mz.ctypes.byref(n), info.ctypes.data)
    assert st == mz.MZ_EINVAL
