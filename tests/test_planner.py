"""Eviction planner (mz_plan_evict) against the reference planner in oracle/
and the workloads' stated plans.  CPU only (host code of the library)."""

import numpy as np
import pytest

import oracle as O
from oracle.planner import eviction_sequence, plan_evict as ref_plan, restore_flops
from paper_2609_01338_amd import mz
from paper_2609_01338_amd import workloads as W

ORDERS = list(mz.ORDERS)
PLACEMENTS = list(mz.PLACEMENTS)


def _cfg(m, n_ctx, n_prompt):
    return mz.make_cfg(m, n_ctx + n_prompt)


def _unit_and_slot(cfg, n_ctx):
    """Device sizes of one weight unit and one KV chunk (layout inputs)."""
    _, _, e = mz.mz_plan_evict(cfg, n_ctx, 0, 0, 1, "backward-out", "all-swap")
    slot = cfg.chunk_tokens * cfg.n_kv_heads * cfg.head_dim * 4
    return int(e["swap_bytes"]), slot


@pytest.mark.parametrize("key,n_kv,n_w,order,placement", [
    ("8b", 3072, 8, "backward-out", "interleave-2-1"),   # 75 % backward-out, 2:1, last 8 weight units
    ("3b", 14 * 32, 0, "backward-out", "all-drop"),       # layers 14-27 dropped
    ("1b", 16 * 8, 0, "forward-out", "all-drop"),         # everything dropped
])
def test_reproduces_the_workload_plans(key, n_kv, n_w, order, placement):
    w = W.WORKLOADS[key]
    cfg = _cfg(w.model, w.n_ctx, w.n_prompt)
    kv, ws, est = mz.mz_plan_evict(cfg, w.n_ctx, w.n_prompt, n_kv, n_w, order, placement)
    p = W.make_plan(w)
    assert np.array_equal(kv, p.kv_state) and np.array_equal(ws, p.w_state)


def test_orders_are_permutations_and_backward_out_is_the_paper_order():
    L, nc = 5, 7
    for order in ORDERS:
        seq = eviction_sequence(L, nc, order, seed=3)
        assert sorted(seq) == [(l, c) for l in range(L) for c in range(nc)]
    assert eviction_sequence(L, nc, "backward-out")[:3] == [(4, 6), (4, 5), (4, 4)]
    assert eviction_sequence(L, nc, "token-aligned")[:3] == [(4, 6), (3, 6), (2, 6)]


SHAPES = [
    # L, d, nq, nkv, hd, ff, C, n_ctx, n_prompt
    (3, 256, 4, 2, 64, 688, 64, 700, 0),
    (4, 512, 8, 2, 64, 1024, 128, 1024, 16),
    (6, 256, 4, 4, 64, 512, 64, 448, 5),
]


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("order", ORDERS)
@pytest.mark.parametrize("placement", PLACEMENTS)
def test_matches_reference_planner(shape, order, placement):
    L, d, nq, nkv, hd, ff, C, n_ctx, n_prompt = shape
    m = W.ModelConfig("t", L, d, nq, nkv, hd, ff, 1024, 1e4, C)
    cfg = _cfg(m, n_ctx, n_prompt)
    unit, slot = _unit_and_slot(cfg, n_ctx)
    nc = (n_ctx + C - 1) // C
    rng = np.random.default_rng(L * 1000 + n_ctx)
    for trial in range(4):
        codec = trial % 2 == 1
        n_kv = int(rng.integers(0, L * nc + 1))
        n_w = int(rng.integers(0, L + 1))
        seed = int(rng.integers(0, 2 ** 63))
        link = float(rng.uniform(1e6, 1e8))          # bytes/s and FLOP/s scaled so both paths matter
        rec = float(rng.uniform(1e9, 1e11))
        kv, ws, est = mz.mz_plan_evict(cfg, n_ctx, n_prompt, n_kv, n_w, order, placement, seed, link, rec,
                                       kv_codec=codec)
        rkv, rws, rlink, rflops = ref_plan(L, d, nq * hd, nkv * hd, ff, C, n_ctx, n_prompt, n_kv, n_w, order,
                                           placement, seed, link, rec, slot, unit, codec=codec)
        assert np.array_equal(kv, rkv), (order, placement, trial)
        assert np.array_equal(ws, rws)
        assert est["swap_bytes"] == rlink
        assert est["restore_flops"] == rflops
        assert int((kv != O.RES).sum()) == n_kv and int((ws != O.RES).sum()) == n_w


def test_estimated_flops_are_the_restore_row_sets():
    """The library's work estimate equals the FLOPs summed over the oracle's
    own R_l / D_l sets for random plans of a workload shape."""
    w = W.WORKLOADS["3b"].scaled(n_layers=5, n_ctx=2048, n_prompt=64)
    m = w.model
    cfg = _cfg(m, w.n_ctx, w.n_prompt)
    for seed in range(3):
        kv, _, est = mz.mz_plan_evict(cfg, w.n_ctx, w.n_prompt, 20 + 7 * seed, 0, "random-out", "all-drop", seed)
        f = restore_flops(m.n_layers, m.d_model, m.dq, m.dkv, m.d_ffn, kv, w.n_ctx, w.n_prompt, m.chunk_tokens)
        assert est["restore_flops"] == f


def test_balanced_beats_fixed_ratio_on_a_fast_link():
    """With the link far cheaper per chunk than recompute, balancing moves
    nearly everything to the link and the predicted restore time drops."""
    w = W.WORKLOADS["8b"]
    cfg = _cfg(w.model, w.n_ctx, w.n_prompt)
    t = {}
    for pl in ("balanced", "interleave-2-1", "all-swap", "all-drop"):
        _, _, e = mz.mz_plan_evict(cfg, w.n_ctx, w.n_prompt, 3072, 8, "backward-out", pl, 0, 56e9, 1.07e15)
        t[pl] = e["pipeline_s"]
        assert e["pipeline_s"] >= max(e["link_s"], e["recompute_s"]) - 1e-12   # a schedule cannot beat either path
    assert t["balanced"] <= min(t.values()) + 1e-12
    assert t["balanced"] < 0.2 * t["interleave-2-1"]


def test_planner_errors():
    w = W.WORKLOADS["tiny"]
    cfg = _cfg(w.model, w.n_ctx, 0)
    with pytest.raises(mz.MzError):
        mz.mz_plan_evict(cfg, w.n_ctx, 0, 10 ** 6, 0)                   # more chunks than exist
    with pytest.raises(mz.MzError):
        mz.mz_plan_evict(cfg, w.n_ctx, 0, 4, 0, "backward-out", "balanced")   # no rates
    with pytest.raises(mz.MzError):
        mz.mz_plan_evict(cfg, w.n_ctx, 0, 4, 99)
