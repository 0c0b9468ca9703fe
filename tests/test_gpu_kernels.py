"""Kernel-level parity on the GPU against the CPU oracle, through the C ABI's
kernel entry points (device buffers allocated with torch).

Tolerances follow from the kernels' arithmetic (u = 2^-11, the f16 unit
roundoff):
 * GEMM: weights d * (q - 8) rounded to f16 (<= u relative) on f16 activations
   (exact inputs), fp32 accumulation: |y - y_ref| <= 2u * sum_k |x_k w_k|
   (+ u |y| for the f16 SwiGLU output).
 * Attention: scores in fp32 from f16 operands (exact products), P rounded to
   f16 (<= u relative), output rounded to f16: |o - o_ref| <= 2u |o_ref| +
   2u max|v|.
 * RMSNorm: fp32 sum of squares, f16 output: 2u relative.
"""

import numpy as np
import pytest

import oracle as O
from paper_2609_01338_amd import mz
from paper_2609_01338_amd import workloads as W
from gpu_util import F16_REL, report, stream, torch_cuda

REL = 2 * F16_REL

pytestmark = pytest.mark.gpu


def _gemm_case(M, N, K, epi, seed, sample_rows=None, n_split=None):
    """n_split: None for mz_q4_gemm, "queued" for mz_q4_gemm_queued (run
    twice from the same initial output on the same queues, which must come
    back zero, and equal to mz_q4_gemm bit for bit), "long-k" for
    mz_q4_gemm_ex with the restore's 64 MiB workspace on a shape it splits
    over K as 256-row tiles, else mz_q4_gemm_split with that many K splits
    ("auto": the restore's choice)."""
    torch = torch_cuda()
    rng = np.random.default_rng(seed)
    report("gemm", M=M, N=N, K=K, epi=epi, seed=seed, n_split=n_split)
    if sample_rows is not None:   # checked on the host: the gather below must stay in bounds
        assert 0 <= int(np.min(sample_rows)) and int(np.max(sample_rows)) < M, "sample rows out of range"
    if epi == 2:
        g = W.encode_q4_0((rng.standard_normal((N, K)) * 0.02).astype(np.float32))
        u = W.encode_q4_0((rng.standard_normal((N, K)) * 0.02).astype(np.float32))
        packed = mz.mz_q4_gemm_pack(g, N, K, w_up=u)
        n_pad = 2 * ((N + 127) // 128 * 128)
    else:
        raw = W.encode_q4_0((rng.standard_normal((N, K)) * 0.02).astype(np.float32))
        packed = mz.mz_q4_gemm_pack(raw, N, K)
        n_pad = (N + 255) // 256 * 256
    gen = torch.Generator(device="cuda").manual_seed(seed)
    x = torch.randn(M, K, device="cuda", generator=gen).to(torch.float16)
    w = torch.from_numpy(packed).cuda()
    if epi == 2:
        y = torch.zeros(M, n_pad // 2, device="cuda", dtype=torch.float16)
    else:
        y = torch.randn(M, n_pad, device="cuda", generator=gen) if epi == 1 else \
            torch.zeros(M, n_pad, device="cuda")
    y0 = y.float().cpu().numpy().astype(np.float64)
    if n_split is None:
        mz.mz_q4_gemm(x.data_ptr(), M, n_pad, K, w.data_ptr(), epi, y.data_ptr(), stream())
    elif n_split == "queued":
        y_init = y.clone()
        mz.mz_q4_gemm(x.data_ptr(), M, n_pad, K, w.data_ptr(), epi, y.data_ptr(), stream())
        plain = y.clone()
        queues = torch.zeros(16, device="cuda", dtype=torch.int32)
        for rep in range(2):
            y.copy_(y_init)
            mz.mz_q4_gemm_queued(x.data_ptr(), M, n_pad, K, w.data_ptr(), epi, y.data_ptr(), queues.data_ptr(),
                                 stream())
            torch.cuda.synchronize()
            assert int(queues.abs().sum()) == 0, "work queues not left at zero"
            assert torch.equal(y.view(torch.uint8), plain.view(torch.uint8)), "queued != mz_q4_gemm"
    elif n_split == "long-k":
        wsb = 64 << 20
        ns = mz.mz_q4_gemm_long_k_splits(M, n_pad, K, wsb)
        report("  long-K splits", n_split=ns)
        assert ns > 1, "shape outside the long-K split rule"
        ws = torch.full((wsb // 4,), float("nan"), device="cuda")      # stale partials must not leak in
        mz.mz_q4_gemm_ex(x.data_ptr(), M, n_pad, K, w.data_ptr(), epi, y.data_ptr(), stream(),
                         workspace=ws.data_ptr(), workspace_bytes=wsb)
    else:
        if n_split == "auto":
            n_split = mz.mz_q4_gemm_auto_splits(M, n_pad, K, 64 << 20)
            report("  auto splits", n_split=n_split)
        wsb = mz.mz_q4_gemm_split_workspace_bytes(M, n_pad, n_split)
        ws = torch.full((wsb // 4,), float("nan"), device="cuda")      # stale partials must not leak in
        mz.mz_q4_gemm_split(x.data_ptr(), M, n_pad, K, w.data_ptr(), epi, y.data_ptr(), n_split, ws.data_ptr(),
                            wsb, stream())
    torch.cuda.synchronize()
    rows = np.arange(M) if sample_rows is None else sample_rows
    xs = x[torch.from_numpy(rows).cuda()].float().cpu().numpy().astype(np.float64)
    ys = y.float().cpu().numpy()[rows].astype(np.float64)
    if epi == 2:
        G = O.q4_0_decode(g.reshape(-1), N, K)
        U = O.q4_0_decode(u.reshape(-1), N, K)
        gr, ur = xs @ G.T, xs @ U.T
        bg = REL * (np.abs(xs) @ np.abs(G).T) + 1e-6
        bu = REL * (np.abs(xs) @ np.abs(U).T) + 1e-6
        ref = O.silu(gr) * ur
        bound = 1.1 * bg * (np.abs(ur) + bu) + np.abs(O.silu(gr)) * bu + REL * np.abs(ref) + 1e-6
        got = ys[:, :N]
        assert np.all(ys[:, N:] == 0)          # padded gate/up columns give silu(0) * 0
    else:
        Wd = O.q4_0_decode(raw.reshape(-1), N, K)
        ref = xs @ Wd.T + (y0[rows, :N] if epi == 1 else 0.0)
        bound = REL * (np.abs(xs) @ np.abs(Wd).T) + 1e-5 * (1 + np.abs(ref))
        got = ys[:, :N]
    err = np.abs(got - ref)
    report("  err", max=float(err.max()), worst_ratio=float((err / bound).max()))
    assert np.all(err <= bound)


@pytest.mark.parametrize("M,N,K,epi", [
    (1, 128, 64, 0), (200, 256, 128, 0), (333, 512, 704, 0), (129, 384, 256, 1),
    (77, 688, 256, 2), (300, 1408, 256, 2)])
def test_gemm_small(M, N, K, epi):
    _gemm_case(M, N, K, epi, seed=M + N + K)


@pytest.mark.parametrize("M,N,K,epi", [
    (1, 256, 640, 0), (5, 512, 1024, 1), (64, 384, 960, 2), (129, 1024, 4096, 1), (200, 688, 512, 2),
    (1, 1408, 2048, 2), (33, 256, 4096, 0)])
def test_gemm_split(M, N, K, epi):
    """Split-K against the exact product: splits that divide the K steps,
    ragged last splits, one step per split, and the restore's choice."""
    nk = K // 64
    for ns in sorted({2, 3, nk, "auto"} - {1}, key=str):
        if ns != "auto" and ns > nk:
            continue
        _gemm_case(M, N, K, epi, seed=M + N + K, n_split=ns)


@pytest.mark.parametrize("M,N,K,epi", [(2048, 2048, 8192, 1), (2000, 2048, 8192, 0), (2048, 2048, 4096, 0),
                                       (2048, 1024, 8192, 2)])
def test_gemm_long_k_split(M, N, K, epi):
    """Products with too few 256-row tiles for the chip but a long K range,
    as the restore launches them (with its workspace): 256-row tiles split
    over K.  The 1B down projection (4 splits of 32 K steps), a ragged last
    row tile, 16 steps per split, and the SwiGLU epilogue, against the exact
    product on one row in every 64-row tile."""
    _gemm_case(M, N, K, epi, seed=M + N + K + 5, sample_rows=_tile_rows(M, 64, M + K), n_split="long-k")


@pytest.mark.parametrize("M", [1, 129])
def test_gemm_split_8b_layer(M):
    """The 8B projections at a decode step (1 row) and a 128-token prompt
    (129 rows), with the restore's split choice."""
    m = W.WORKLOADS["8b"].model
    ffp = (m.d_ffn + 127) // 128 * 128
    for i, (N, K, epi) in enumerate([(m.dq, m.d_model, 0), (2 * m.dkv, m.d_model, 0), (m.d_model, m.dq, 1),
                                     (m.d_ffn, m.d_model, 2), (m.d_model, ffp, 1)]):
        _gemm_case(M, N, K, epi, seed=300 + i, n_split="auto")


def test_gemm_split_validation():
    torch_cuda()
    with pytest.raises(mz.MzError):
        mz.mz_q4_gemm_split(1, 4, 256, 640, 1, 0, 1, 2, 1, 100, None)     # workspace too small
    with pytest.raises(mz.MzError):
        mz.mz_q4_gemm_split(1, 4, 256, 640, 1, 0, 1, 0, 1, 1 << 20, None)  # n_split 0
    with pytest.raises(mz.MzError):
        mz.mz_q4_gemm_queued(1, 4, 256, 640, 1, 0, 1, 0, None)            # no work queues
    assert mz.mz_q4_gemm_auto_splits(32896, 4096, 4096, 64 << 20) == 1
    assert mz.mz_q4_gemm_auto_splits(1, 4096, 14336, 64 << 20) > 8


def _layer_gemms(key):
    w = W.WORKLOADS[key]
    m = w.model
    M = w.n_ctx + w.n_prompt
    ffp = (m.d_ffn + 127) // 128 * 128
    return [(M, m.dq + 2 * m.dkv, m.d_model, 0), (M, m.d_model, m.dq, 1),
            (M, m.d_ffn, m.d_model, 2), (M, m.d_model, ffp, 1)]


def _tile_rows(M, tile, seed):
    """One row in every `tile`-row tile (at a seeded offset inside it), the
    first and last rows, and both sides of the last whole 256-row tile."""
    rng = np.random.default_rng(seed)
    starts = np.arange(0, M, tile)
    rows = np.minimum(starts + rng.integers(0, tile, starts.size), M - 1)
    edge = [r for r in (M // 256 * 256 - 1, M // 256 * 256) if 0 <= r < M]
    return np.unique(np.concatenate([rows, [0, M - 1], edge])).astype(np.int64)


@pytest.mark.parametrize("key", ["tiny", "1b", "3b", "1p5b", "8b"])
def test_gemm_full_layer_shapes(key):
    """Every projection of the workload at its full row count (the launch the
    benchmark times), checked on one row in every 64-row tile (so in every
    256- and 64-row tile of either launch form) including the ragged tail and
    both sides of the row where whole 256-row tiles end."""
    for i, (M, N, K, epi) in enumerate(_layer_gemms(key)):
        _gemm_case(M, N, K, epi, seed=100 + i, sample_rows=_tile_rows(M, 64, i), n_split="queued")


def _rope_table(max_pos, hd, theta):
    """(cos, sin) of p * theta^(-2i/hd) in fp64, stored as fp32 pairs [max_pos][hd/2]."""
    i = np.arange(hd // 2, dtype=np.float64)
    ang = np.arange(max_pos, dtype=np.float64)[:, None] * theta ** (-2.0 * i / hd)[None, :]
    return np.stack([np.cos(ang), np.sin(ang)], axis=-1).astype(np.float32)


@pytest.mark.parametrize("key", ["1b", "3b", "1p5b", "8b"])
def test_gemm_restore_launches(key):
    """The projections as the restore launches them (mz_q4_gemm_ex), at the
    workload's full row count: with the runtime's 64 MiB workspace, so the
    rows after the last whole 256-row tile run split over K where their tiles
    alone would leave the chip idle; through a row list (a ragged subset of the
    activation rows, as the restore passes R_l / D_l); with the work queues;
    and with the rotary epilogues (queries to f16; keys and values into chunk
    slots).  Against the exact product (and the oracle's rotary embedding) on
    one row in every 64-row tile and both sides of the last whole 256-row
    tile; rows in whole 256-row tiles bit-equal to mz_q4_gemm's."""
    torch = torch_cuda()
    w = W.WORKLOADS[key]
    m = w.model
    S = w.n_ctx + w.n_prompt
    d, hd, C = m.d_model, m.head_dim, m.chunk_tokens
    rng = np.random.default_rng(17)
    gen = torch.Generator(device="cuda").manual_seed(17)
    X = torch.randn(S, d, device="cuda", generator=gen).to(torch.float16)
    Xh = X.float().cpu().numpy().astype(np.float64)
    ws_bytes = 64 << 20
    ws = torch.full((ws_bytes // 4,), float("nan"), device="cuda")
    queues = torch.zeros(16, device="cuda", dtype=torch.int32)
    cs = torch.from_numpy(_rope_table(S, hd, m.rope_theta)).cuda()
    # a ragged row list: every row of a random half of the chunks, then the prompt
    keep = rng.random(w.n_chunks) < 0.5
    sub = np.array([p for p in range(S) if p >= w.n_ctx or keep[p // C]], np.int32)
    d_sub = torch.from_numpy(sub).cuda()
    for rows_name, M, arow, pos_np in (("all", S, None, np.arange(S, dtype=np.int32)), ("list", sub.size, sub, sub)):
        d_pos = torch.from_numpy(np.ascontiguousarray(pos_np)).cuda()
        xr = Xh if arow is None else Xh[arow]
        ar_ptr = 0 if arow is None else d_sub.data_ptr()
        check = _tile_rows(M, 64, M)
        full = M // 256 * 256
        # queries, rotated
        raw = W.encode_q4_0((rng.standard_normal((m.dq, d)) * 0.02).astype(np.float32))
        Wm = O.q4_0_decode(raw.reshape(-1), m.dq, d)
        n_pad = (m.dq + 255) // 256 * 256
        wdev = torch.from_numpy(mz.mz_q4_gemm_pack(raw, m.dq, d)).cuda()
        yq = torch.full((M, m.dq), float("nan"), device="cuda", dtype=torch.float16)
        report("restore launch", workload=key, rows=rows_name, M=M, proj="q-rope")
        mz.mz_q4_gemm_ex(X.data_ptr(), M, n_pad, d, wdev.data_ptr(), 4, yq.data_ptr(), stream(), a_rows=ar_ptr,
                         workspace=ws.data_ptr(), workspace_bytes=ws_bytes, pos=d_pos.data_ptr(),
                         rope_cs=cs.data_ptr(), head_dim=hd, n_valid=m.dq)
        torch.cuda.synchronize()
        xs = xr[check]
        prod = xs @ Wm.T
        b = REL * (np.abs(xs) @ np.abs(Wm).T) + 1e-6
        ref = O.rope(prod.reshape(-1, m.n_q_heads, hd), pos_np[check], m.rope_theta).reshape(-1, m.dq)
        bh = b.reshape(-1, m.n_q_heads, hd)
        bound = (bh + np.concatenate([bh[..., hd // 2:], bh[..., :hd // 2]], -1)).reshape(-1, m.dq)
        bound = bound + F16_REL * np.abs(ref) + 2.0 ** -22 * np.abs(prod).max()
        got = yq.float().cpu().numpy()[check].astype(np.float64)
        err = np.abs(got - ref)
        report("  err", max=float(err.max()), worst_ratio=float((err / bound).max()))
        assert np.all(err <= bound)
        # keys and values into chunk slots
        rk = W.encode_q4_0((rng.standard_normal((m.dkv, d)) * 0.02).astype(np.float32))
        rv = W.encode_q4_0((rng.standard_normal((m.dkv, d)) * 0.02).astype(np.float32))
        Wk, Wv = O.q4_0_decode(rk.reshape(-1), m.dkv, d), O.q4_0_decode(rv.reshape(-1), m.dkv, d)
        n_kv = 2 * m.dkv
        wdev = torch.from_numpy(mz.mz_q4_gemm_pack(np.concatenate([rk, rv]), n_kv, d)).cuda()
        n_slots = (S + C - 1) // C + 1
        slot_bytes = C * m.dkv * 4
        perm = rng.permutation(n_slots)[: (S + C - 1) // C]
        kv_off = (perm[pos_np // C].astype(np.int64) * slot_bytes + (pos_np % C).astype(np.int64) * m.dkv * 2)
        slab = torch.full((n_slots * slot_bytes // 2,), float("nan"), device="cuda", dtype=torch.float16)
        d_off = torch.from_numpy(kv_off).cuda()
        report("restore launch", workload=key, rows=rows_name, M=M, proj="kv-rope-slots")
        mz.mz_q4_gemm_ex(X.data_ptr(), M, (n_kv + 255) // 256 * 256, d, wdev.data_ptr(), 5, 0, stream(),
                         a_rows=ar_ptr, workspace=ws.data_ptr(), workspace_bytes=ws_bytes, pos=d_pos.data_ptr(),
                         rope_cs=cs.data_ptr(), kv_off=d_off.data_ptr(), slab=slab.data_ptr(), head_dim=hd,
                         n_valid=n_kv, chunk_tokens=C)
        torch.cuda.synchronize()
        sl = slab.view(torch.uint8).cpu().numpy()
        pk, pv = xs @ Wk.T, xs @ Wv.T
        bk = REL * (np.abs(xs) @ np.abs(Wk).T) + 1e-6
        bv = REL * (np.abs(xs) @ np.abs(Wv).T) + 1e-6
        kref = O.rope(pk.reshape(-1, m.n_kv_heads, hd), pos_np[check], m.rope_theta).reshape(-1, m.dkv)
        bkh = bk.reshape(-1, m.n_kv_heads, hd)
        kb = (bkh + np.concatenate([bkh[..., hd // 2:], bkh[..., :hd // 2]], -1)).reshape(-1, m.dkv)
        kb = kb + F16_REL * np.abs(kref) + 2.0 ** -22 * np.abs(pk).max()
        vb = bv + F16_REL * np.abs(pv)
        for j, r in enumerate(check):
            off = int(kv_off[r])
            kg = sl[off:off + m.dkv * 2].view(np.float16).astype(np.float64)
            base = off - int(pos_np[r] % C) * m.dkv * 2 + C * m.dkv * 2
            vt = sl[base:base + m.dkv * C * 2].view(np.float16).reshape(m.dkv, C)[:, pos_np[r] % C]
            assert np.all(np.abs(kg - kref[j]) <= kb[j]), (key, rows_name, int(r), "K")
            assert np.all(np.abs(vt.astype(np.float64) - pv[j]) <= vb[j]), (key, rows_name, int(r), "V")
        # plain epilogues (store, residual add, SwiGLU) with queues and workspace,
        # against mz_q4_gemm bit for bit on whole 256-row tiles
        for i, (N, K, epi) in enumerate([(m.d_model, m.dq, 1), (m.d_ffn, m.d_model, 2)]):
            if K != d:
                continue           # the activation rows are [S][d]
            if epi == 2:
                g_ = W.encode_q4_0((rng.standard_normal((N, K)) * 0.02).astype(np.float32))
                u_ = W.encode_q4_0((rng.standard_normal((N, K)) * 0.02).astype(np.float32))
                wdev = torch.from_numpy(mz.mz_q4_gemm_pack(g_, N, K, w_up=u_)).cuda()
                n_pad = 2 * ((N + 127) // 128 * 128)
                y1 = torch.zeros(M, n_pad // 2, device="cuda", dtype=torch.float16)
            else:
                raw = W.encode_q4_0((rng.standard_normal((N, K)) * 0.02).astype(np.float32))
                wdev = torch.from_numpy(mz.mz_q4_gemm_pack(raw, N, K)).cuda()
                n_pad = (N + 255) // 256 * 256
                y1 = torch.randn(M, n_pad, device="cuda", generator=gen)
            y0 = y1.clone()
            xg = X if arow is None else X[d_sub.long()].contiguous()
            report("restore launch", workload=key, rows=rows_name, M=M, proj=f"epi{epi}")
            mz.mz_q4_gemm_ex(X.data_ptr(), M, n_pad, K, wdev.data_ptr(), epi, y1.data_ptr(), stream(), a_rows=ar_ptr,
                             work_queues=queues.data_ptr(), workspace=ws.data_ptr(), workspace_bytes=ws_bytes)
            y2 = y0.clone()
            mz.mz_q4_gemm(xg.data_ptr(), M, n_pad, K, wdev.data_ptr(), epi, y2.data_ptr(), stream())
            torch.cuda.synchronize()
            assert int(queues.abs().sum()) == 0
            assert torch.equal(y1[:full].view(torch.uint8), y2[:full].view(torch.uint8)), (key, rows_name, epi)
            a1 = y1[full:].float().cpu().numpy().astype(np.float64)
            a2 = y2[full:].float().cpu().numpy().astype(np.float64)
            if a1.size:
                scale = np.abs(a2).max() + 1e-3
                assert np.abs(a1 - a2).max() <= 4 * F16_REL * scale, (key, rows_name, epi)


def _single_row_shapes(key):
    m = W.WORKLOADS[key].model
    ffp = (m.d_ffn + 127) // 128 * 128      # the SwiGLU output width, as the down projection reads it
    return [("q-rope", m.dq, m.d_model, 4), ("kv-rope-slots", 2 * m.dkv, m.d_model, 5),
            ("q-store", m.dq, m.d_model, 0), ("o-add", m.d_model, m.dq, 1),
            ("gateup-swiglu", m.d_ffn, m.d_model, 2), ("down-add", m.d_model, ffp, 1)]


@pytest.mark.parametrize("key", ["tiny", "1b", "3b", "1p5b", "8b"])
def test_gemv_single_row(key):
    """mz_q4_gemv, the one-launch single-row product (decode steps), for every
    projection of the workload at its full shape, with each epilogue the
    runtime gives it: against the exact product of the decoded weights (and
    the oracle's rotary embedding) on every output column, for a row picked
    from a matrix through a_rows; the RMSNorm-forming variant against the
    same product of mz_rmsnorm's output, bit for bit."""
    torch = torch_cuda()
    w = W.WORKLOADS[key]
    m = w.model
    hd, C = m.head_dim, m.chunk_tokens
    rng = np.random.default_rng(23)
    gen = torch.Generator(device="cuda").manual_seed(23)
    n_rows = 5
    row = 3
    d_row = torch.tensor([row], device="cuda", dtype=torch.int32)
    p = int(w.n_ctx + w.n_prompt - 1)                 # the position of a decode row
    cs = torch.from_numpy(_rope_table(p + 1, hd, m.rope_theta)).cuda()
    d_pos = torch.tensor([p], device="cuda", dtype=torch.int32)
    for name, N, K, epi in _single_row_shapes(key):
        report("gemv", workload=key, proj=name, N=N, K=K, epi=epi)
        X = torch.randn(n_rows, K, device="cuda", generator=gen).to(torch.float16)
        xs = X[row].float().cpu().numpy().astype(np.float64)[None, :]
        if epi == 2:
            g_ = W.encode_q4_0((rng.standard_normal((N, K)) * 0.02).astype(np.float32))
            u_ = W.encode_q4_0((rng.standard_normal((N, K)) * 0.02).astype(np.float32))
            wdev = torch.from_numpy(mz.mz_q4_gemm_pack(g_, N, K, w_up=u_)).cuda()
            n_pad = 2 * ((N + 127) // 128 * 128)
            G, U = O.q4_0_decode(g_.reshape(-1), N, K), O.q4_0_decode(u_.reshape(-1), N, K)
        elif epi == 5:
            half_n = N // 2
            rk = W.encode_q4_0((rng.standard_normal((half_n, K)) * 0.02).astype(np.float32))
            rv = W.encode_q4_0((rng.standard_normal((half_n, K)) * 0.02).astype(np.float32))
            wdev = torch.from_numpy(mz.mz_q4_gemm_pack(np.concatenate([rk, rv]), N, K)).cuda()
            n_pad = (N + 255) // 256 * 256
            Wk, Wv = O.q4_0_decode(rk.reshape(-1), half_n, K), O.q4_0_decode(rv.reshape(-1), half_n, K)
        else:
            raw = W.encode_q4_0((rng.standard_normal((N, K)) * 0.02).astype(np.float32))
            wdev = torch.from_numpy(mz.mz_q4_gemm_pack(raw, N, K)).cuda()
            n_pad = (N + 255) // 256 * 256
            Wm = O.q4_0_decode(raw.reshape(-1), N, K)

        def run(x_ptr, h_ptr, out):
            kw = dict(a_rows=d_row.data_ptr(), h_norm=h_ptr, eps=float(m.rms_eps))
            if epi == 4:
                kw.update(pos=d_pos.data_ptr(), rope_cs=cs.data_ptr(), head_dim=hd, n_valid=N)
            if epi == 5:
                kw.update(pos=d_pos.data_ptr(), rope_cs=cs.data_ptr(), kv_off=d_off.data_ptr(),
                          slab=out.data_ptr(), head_dim=hd, n_valid=N, chunk_tokens=C)
            mz.mz_q4_gemv(x_ptr, K, wdev.data_ptr(), n_pad, epi, 0 if epi == 5 else out.data_ptr(), stream(),
                          **kw)

        if epi == 5:
            slot_bytes = C * (N // 2) * 4
            slot, pc = 2, p % C
            out = torch.full((4 * slot_bytes // 2,), float("nan"), device="cuda", dtype=torch.float16)
            d_off = torch.tensor([slot * slot_bytes + pc * (N // 2) * 2], device="cuda", dtype=torch.int64)
        elif epi == 4:
            out = torch.full((1, N), float("nan"), device="cuda", dtype=torch.float16)
        elif epi == 2:
            out = torch.full((1, n_pad // 2), float("nan"), device="cuda", dtype=torch.float16)
        elif epi == 1:
            out = torch.randn(1, n_pad, device="cuda", generator=gen)
        else:
            out = torch.full((1, n_pad), float("nan"), device="cuda")
        out0 = out.clone()
        run(X.data_ptr(), 0, out)
        torch.cuda.synchronize()
        if epi == 4:
            prod = xs @ Wm.T
            b = REL * (np.abs(xs) @ np.abs(Wm).T) + 1e-6
            ref = O.rope(prod.reshape(1, m.n_q_heads, hd), np.array([p]), m.rope_theta).reshape(1, N)
            bh = b.reshape(1, m.n_q_heads, hd)
            bound = (bh + np.concatenate([bh[..., hd // 2:], bh[..., :hd // 2]], -1)).reshape(1, N)
            bound = bound + F16_REL * np.abs(ref) + 2.0 ** -22 * np.abs(prod).max()
            got = out.float().cpu().numpy().astype(np.float64)
        elif epi == 5:
            dkv = N // 2
            pk, pv = xs @ Wk.T, xs @ Wv.T
            bk = REL * (np.abs(xs) @ np.abs(Wk).T) + 1e-6
            bv = REL * (np.abs(xs) @ np.abs(Wv).T) + 1e-6
            kref = O.rope(pk.reshape(1, m.n_kv_heads, hd), np.array([p]), m.rope_theta).reshape(1, dkv)
            bkh = bk.reshape(1, m.n_kv_heads, hd)
            kb = (bkh + np.concatenate([bkh[..., hd // 2:], bkh[..., :hd // 2]], -1)).reshape(1, dkv)
            kb = kb + F16_REL * np.abs(kref) + 2.0 ** -22 * np.abs(pk).max()
            sl = out.view(torch.uint8).cpu().numpy()
            off = slot * slot_bytes + pc * dkv * 2
            kg = sl[off:off + dkv * 2].view(np.float16).astype(np.float64)[None, :]
            base = slot * slot_bytes + C * dkv * 2
            vt = sl[base:base + dkv * C * 2].view(np.float16).reshape(dkv, C)[:, pc].astype(np.float64)[None, :]
            got = np.concatenate([kg, vt], 1)
            ref = np.concatenate([kref, pv], 1)
            bound = np.concatenate([kb, bv + F16_REL * np.abs(pv)], 1)
            # nothing else of the slab was written
            touched = np.zeros(sl.size // 2, bool)
            touched[off // 2: off // 2 + dkv] = True
            touched[base // 2 + np.arange(dkv) * C + pc] = True
            assert np.all(np.isnan(out.float().cpu().numpy()[~touched]))
        elif epi == 2:
            gr, ur = xs @ G.T, xs @ U.T
            bg = REL * (np.abs(xs) @ np.abs(G).T) + 1e-6
            bu = REL * (np.abs(xs) @ np.abs(U).T) + 1e-6
            ref = O.silu(gr) * ur
            bound = 1.1 * bg * (np.abs(ur) + bu) + np.abs(O.silu(gr)) * bu + REL * np.abs(ref) + 1e-6
            ys = out.float().cpu().numpy().astype(np.float64)
            got = ys[:, :N]
            assert np.all(ys[:, N:] == 0)          # padded gate/up columns give silu(0) * 0
        else:
            ref = xs @ Wm.T + (out0.cpu().numpy().astype(np.float64)[:, :N] if epi == 1 else 0.0)
            bound = REL * (np.abs(xs) @ np.abs(Wm).T) + 1e-5 * (1 + np.abs(ref))
            got = out.cpu().numpy().astype(np.float64)[:, :N]
        err = np.abs(got - ref)
        report("  err", max=float(err.max()), worst_ratio=float((err / bound).max()))
        assert np.all(err <= bound), (key, name)
        # the RMSNorm-forming variant: the same bits as the product of mz_rmsnorm's rows
        if K == m.d_model:
            H = torch.randn(n_rows, K, device="cuda", generator=gen) * 3.0
            Xn = torch.empty(n_rows, K, device="cuda", dtype=torch.float16)
            mz.mz_rmsnorm(H.data_ptr(), n_rows, K, float(m.rms_eps), Xn.data_ptr(), stream())
            o1, o2 = out0.clone(), out0.clone()
            if epi == 5:
                o1.fill_(float("nan"))
                o2.fill_(float("nan"))
            run(Xn.data_ptr(), 0, o1)
            run(0, H.data_ptr(), o2)
            torch.cuda.synchronize()
            assert torch.equal(o1.view(torch.uint8), o2.view(torch.uint8)), (key, name, "norm in gemv")


def test_gemv_validation():
    torch = torch_cuda()
    x = torch.zeros(1, 256, device="cuda", dtype=torch.float16)
    w = torch.zeros(mz.mz_q4_gemm_packed_bytes(256, 256), device="cuda", dtype=torch.uint8)
    y = torch.zeros(1, 256, device="cuda")
    bad = [dict(k=256, n_pad=100, epi=0), dict(k=100, n_pad=256, epi=0), dict(k=16448, n_pad=256, epi=0),
           dict(k=256, n_pad=256, epi=3), dict(k=256, n_pad=256, epi=4)]
    for b in bad:
        with pytest.raises(mz.MzError):
            mz.mz_q4_gemv(x.data_ptr(), b["k"], w.data_ptr(), b["n_pad"], b["epi"], y.data_ptr(), stream())
    with pytest.raises(mz.MzError):
        mz.mz_q4_gemv(x.data_ptr(), 256, w.data_ptr(), 256, 0, y.data_ptr(), stream(), h_norm=y.data_ptr(),
                      eps=-1.0)


@pytest.mark.parametrize("M,N,K,epi", [
    (20000, 14336, 128, 0), (16640, 16384, 64, 1), (20000, 7168, 128, 2), (33000, 8192, 64, 1),
    (1000, 2048, 512, 0), (9000, 4096, 512, 1), (300, 512, 128, 1)])
def test_gemm_queued(M, N, K, epi):
    """mz_q4_gemm_queued for every plain epilogue: launches of at least 16
    rounds (4096 and more 256-row tiles) take the work queues, with and
    without a ragged remainder of 64-row tiles; shorter ones run one
    workgroup per tile.  Against the exact product on sampled rows and
    bit-equal to mz_q4_gemm."""
    rows = None
    if M > 4000:
        rng = np.random.default_rng(M)
        rows = np.unique(np.concatenate([rng.choice(M, 40, replace=False),
                                         [0, M // 256 * 256 - 1, M // 256 * 256, M - 1]]))
        rows = rows[rows < M]   # M // 256 * 256 is M itself when M is a multiple of 256
    _gemm_case(M, N, K, epi, seed=M + 7, sample_rows=rows, n_split="queued")


def _attn_case(nq, nkv, hd, C, S, qpos, seed, sample=None, n_split=None, n_table=None):
    """n_split: None for mz_attention, "queued" for mz_attention_queued (run
    twice on the same queues, which must come back zero, and equal to
    mz_attention bit for bit), else mz_attention_split with that many key
    splits ("auto": the restore's choice)."""
    torch = torch_cuda()
    report("attention", nq=nq, nkv=nkv, hd=hd, C=C, S=S, m=len(qpos), seed=seed, n_split=n_split)
    if sample is not None:
        assert 0 <= int(np.min(sample)) and int(np.max(sample)) < len(qpos), "sample rows out of range"
    rng = np.random.default_rng(seed)
    dkv = nkv * hd
    nch = (S + C - 1) // C
    n_slots = nch + 3
    table = rng.permutation(n_slots)[:nch].astype(np.int32)
    K = rng.standard_normal((S, dkv)).astype(np.float16)
    V = rng.standard_normal((S, dkv)).astype(np.float16)
    # slot: K [C][dkv] token-major, then V^T [dkv][C]; unused rows are NaN
    kpart = np.full((n_slots, C, dkv), np.nan, np.float16)
    vpart = np.full((n_slots, dkv, C), np.nan, np.float16)
    for c in range(nch):
        n = min(C, S - c * C)
        kpart[table[c], :n] = K[c * C:c * C + n]
        vpart[table[c], :, :n] = V[c * C:c * C + n].T
    slab = np.concatenate([kpart.reshape(n_slots, -1), vpart.reshape(n_slots, -1)], axis=1)
    if n_table is not None:
        # a longer table than the keys need (entries past them name slot 0)
        table = np.concatenate([table, np.zeros(n_table - nch, np.int32)])
        nch = n_table
    qpos = np.asarray(qpos, np.int32)
    M = qpos.size
    q = (rng.standard_normal((M, nq, hd)) * 1.0).astype(np.float16)
    d_q = torch.from_numpy(q).cuda()
    d_pos = torch.from_numpy(qpos).cuda()
    d_slab = torch.from_numpy(slab).cuda()
    d_tab = torch.from_numpy(table).cuda()
    out = torch.empty(M, nq * hd, device="cuda", dtype=torch.float16)
    max_pos = int(qpos[-1])
    if n_split is None:
        mz.mz_attention(d_q.data_ptr(), d_pos.data_ptr(), M, d_slab.data_ptr(), d_tab.data_ptr(), nch, C,
                        nq, nkv, hd, out.data_ptr(), stream())
    elif n_split == "queued":
        queues = torch.zeros(16, device="cuda", dtype=torch.int32)
        plain = torch.empty_like(out)
        mz.mz_attention(d_q.data_ptr(), d_pos.data_ptr(), M, d_slab.data_ptr(), d_tab.data_ptr(), nch, C,
                        nq, nkv, hd, plain.data_ptr(), stream())
        for rep in range(2):
            out.fill_(float("nan"))
            mz.mz_attention_queued(d_q.data_ptr(), d_pos.data_ptr(), M, d_slab.data_ptr(), d_tab.data_ptr(), nch,
                                   C, nq, nkv, hd, out.data_ptr(), queues.data_ptr(), stream())
            torch.cuda.synchronize()
            assert int(queues.abs().sum()) == 0, "work queues not left at zero"
            assert torch.equal(out.view(torch.int16), plain.view(torch.int16)), "queued != mz_attention"
    else:
        if n_split == "auto":
            n_split = mz.mz_attention_auto_splits(M, max_pos, nq, nkv, hd, 64 << 20)
            report("  auto splits", n_split=n_split)
        wsb = mz.mz_attention_split_workspace_bytes(M, nq, hd, n_split)
        ws = torch.empty(wsb, device="cuda", dtype=torch.uint8)
        mz.mz_attention_split(d_q.data_ptr(), d_pos.data_ptr(), M, max_pos, d_slab.data_ptr(), d_tab.data_ptr(),
                              nch, C, nq, nkv, hd, n_split, ws.data_ptr(), wsb, out.data_ptr(), stream())
    torch.cuda.synchronize()
    got = out.float().cpu().numpy().reshape(M, nq, hd).astype(np.float64)
    rows = np.arange(M) if sample is None else sample
    ref = O.causal_gqa_attention(q[rows].astype(np.float64), qpos[rows],
                                 K.astype(np.float64).reshape(S, nkv, hd),
                                 V.astype(np.float64).reshape(S, nkv, hd))
    g = got[rows]
    bound = REL * np.abs(ref) + 2.0 ** -10 * float(np.abs(V).max())
    if n_split is not None:
        # each split's normalised output is a convex combination of V rows,
        # rounded to f16 (half an ulp: 2^-11 max|V|); the merge is again a
        # convex combination of those
        bound = bound + 2.0 ** -11 * float(np.abs(V).max())
    err = np.abs(g - ref)
    report("  err", max=float(err.max()), worst_ratio=float((err / bound).max()))
    assert np.all(np.isfinite(g))
    assert np.all(err <= bound)


@pytest.mark.parametrize("nq,nkv,hd,C,S", [
    (4, 2, 64, 16, 128), (4, 2, 64, 16, 117), (32, 8, 64, 256, 600), (24, 8, 128, 256, 700),
    (12, 2, 128, 256, 530), (32, 8, 128, 256, 400), (8, 8, 128, 64, 200), (6, 1, 64, 32, 90),
    (4, 4, 128, 8, 77), (10, 2, 64, 64, 450), (14, 2, 128, 128, 600), (16, 2, 64, 32, 333)])
def test_attention_small(nq, nkv, hd, C, S):
    """Query-head groups of 1-8 (so every wave map: G heads x 8/G row groups,
    2 heads x 4 for G = 6, one head x 8 for G = 3, 5, 7), dense, gappy, first
    and last query rows, against the exact definition."""
    rng = np.random.default_rng(S)
    dense = np.arange(S)
    gappy = np.sort(rng.choice(S, max(1, S // 3), replace=False))
    _attn_case(nq, nkv, hd, C, S, dense, seed=1)
    _attn_case(nq, nkv, hd, C, S, gappy, seed=2)
    _attn_case(nq, nkv, hd, C, S, [0], seed=3)
    _attn_case(nq, nkv, hd, C, S, [S - 1], seed=4)


@pytest.mark.parametrize("key", ["1b", "3b", "1p5b", "8b"])
def test_attention_full_context(key):
    """All S query rows of the workload through the work queues (the
    restore's launch), bit-equal to the one-tile-per-workgroup form, and one
    query row (every head, so every KV head) in every 32-row query tile
    checked against the exact definition."""
    w = W.WORKLOADS[key]
    m = w.model
    S = w.n_ctx + w.n_prompt
    _attn_case(m.n_q_heads, m.n_kv_heads, m.head_dim, m.chunk_tokens, S, np.arange(S), seed=5,
               sample=_tile_rows(S, 32, 5), n_split="queued")


def test_attention_full_context_gappy_1p5b():
    """The 1.5B shape (12 query / 2 KV heads, head dim 128) at its full
    16384-token context with gappy query rows: the rows of a seeded 30 % of
    the chunks (a recompute's R_l), through the work queues; one query in
    every 32-row tile checked."""
    w = W.WORKLOADS["1p5b"]
    m = w.model
    S = w.n_ctx
    rng = np.random.default_rng(31)
    keep = rng.random(w.n_chunks) < 0.3
    qpos = np.array([p for p in range(S) if keep[p // m.chunk_tokens] or p == S - 1], np.int32)
    _attn_case(m.n_q_heads, m.n_kv_heads, m.head_dim, m.chunk_tokens, S, qpos, seed=6,
               sample=_tile_rows(qpos.size, 32, 6), n_split="queued")


@pytest.mark.parametrize("nq,nkv,hd,C,S", [
    (32, 8, 128, 256, 3000), (24, 8, 128, 256, 1700), (12, 2, 128, 256, 1030), (16, 4, 64, 64, 900),
    (8, 8, 128, 64, 200), (6, 1, 64, 128, 700), (12, 3, 64, 256, 600), (4, 4, 128, 8, 77)])
def test_attention_queued(nq, nkv, hd, C, S):
    """The work-queue form: 1, 2, 4 and 8 KV heads (queues shared by 8, 4, 2
    and 1 XCDs), more tiles than workgroups and fewer, gappy query rows; 3
    KV heads and 8-token chunks take the one-tile-per-workgroup form."""
    rng = np.random.default_rng(S + 1)
    gappy = np.sort(rng.choice(S, max(1, S // 3), replace=False))
    _attn_case(nq, nkv, hd, C, S, np.arange(S), seed=11, n_split="queued")
    _attn_case(nq, nkv, hd, C, S, gappy, seed=12, n_split="queued")
    _attn_case(nq, nkv, hd, C, S, [S - 1], seed=13, n_split="queued")


def test_attention_max_table():
    """A chunk table of 8192 entries, the most the attention entry points
    take (its stretch for each work item is copied into LDS): the plain, the
    work-queue and the split forms against the exact definition."""
    for n_split in (None, "queued", 4):
        _attn_case(32, 8, 128, 64, 700, np.arange(700), seed=41, n_split=n_split, n_table=8192)


@pytest.mark.parametrize("nq,nkv,hd,C,S", [
    (4, 2, 64, 16, 700), (32, 8, 128, 256, 2000), (24, 8, 128, 256, 1500), (12, 2, 128, 256, 1100),
    (8, 8, 128, 64, 900), (6, 1, 64, 32, 800), (4, 4, 128, 8, 333)])
def test_attention_split(nq, nkv, hd, C, S):
    """Split-key attention against the exact definition: prompt-like tails,
    one row, rows far apart (early rows see no key of the later splits), and
    a row at position 0; 2..64 splits (one tile per split at the top)."""
    rng = np.random.default_rng(S + nq)
    cases = [np.arange(S - 9, S), [S - 1], [3, S // 2, S - 1], np.concatenate([[10], np.arange(S - 70, S)]),
             np.sort(rng.choice(S, 40, replace=False)), [0]]
    for i, qp in enumerate(cases):
        for n_split in (2, 5, "auto", 64):
            _attn_case(nq, nkv, hd, C, S, qp, seed=20 + i, n_split=n_split)


@pytest.mark.parametrize("m", [1, 4, 129])
def test_attention_split_8b_context(m):
    """The 8B layer at its full context (32768 cached + 128 prompt tokens):
    the last m rows, as the restore runs them when nothing before the prompt
    is recomputed, with the restore's split choice; every row checked.  One
    and four rows take the few-column kernel (4 and 16 (row, head) columns
    of a KV head), 129 rows the tiled one."""
    w = W.WORKLOADS["8b"]
    mdl = w.model
    S = w.n_ctx + w.n_prompt
    _attn_case(mdl.n_q_heads, mdl.n_kv_heads, mdl.head_dim, mdl.chunk_tokens, S, np.arange(S - m, S), seed=9,
               n_split="auto")
    if m == 4:   # four rows far apart (different splits hold their last keys)
        _attn_case(mdl.n_q_heads, mdl.n_kv_heads, mdl.head_dim, mdl.chunk_tokens, S,
                   np.array([5, 300, 17000, S - 1]), seed=10, n_split="auto")


def test_attention_split_validation():
    torch_cuda()
    with pytest.raises(mz.MzError):
        mz.mz_attention_split(1, 1, 4, 100, 1, 1, 1, 16, 8, 2, 64, 2, 1, 10, 1)   # table short of max_pos
    with pytest.raises(mz.MzError):
        mz.mz_attention_split(1, 1, 4, 10, 1, 1, 1, 16, 8, 2, 64, 2, 1, 10, 1)    # workspace too small
    with pytest.raises(mz.MzError):
        mz.mz_attention_split(1, 1, 4, 10, 1, 1, 1, 16, 8, 2, 64, 65, 1, 1 << 30, 1)   # more than 64 splits
    with pytest.raises(mz.MzError):
        mz.mz_attention_queued(1, 1, 4, 1, 1, 1, 16, 8, 2, 64, 1, 0, 1)   # no work queues
    assert mz.mz_attention_auto_splits(40000, 40000, 32, 8, 128, 64 << 20) == 1   # the chip is full already
    # one decode row (4 columns per KV head): about one workgroup per CU
    assert 24 <= mz.mz_attention_auto_splits(1, 32895, 32, 8, 128, 64 << 20) <= 32
    assert mz.mz_attention_auto_splits(129, 32895, 32, 8, 128, 64 << 20) > 8


@pytest.mark.parametrize("M,d", [(1, 256), (300, 2048), (77, 4096), (5, 1536), (3, 8196), (2, 12292)])
def test_rmsnorm(M, d):
    torch = torch_cuda()
    rng = np.random.default_rng(M * d)
    h = (rng.standard_normal((M, d)) * 3).astype(np.float32)
    h[0, :] *= 1e-3
    x = torch.empty(M, d, device="cuda", dtype=torch.float16)
    dh = torch.from_numpy(h).cuda()
    mz.mz_rmsnorm(dh.data_ptr(), M, d, 1e-5, x.data_ptr(), stream())
    torch.cuda.synchronize()
    ref = O.rmsnorm(h.astype(np.float64), 1e-5)
    got = x.float().cpu().numpy()
    assert np.all(np.abs(got - ref) <= REL * np.abs(ref) + 1e-6)


def test_kernel_entry_validation():
    torch_cuda()
    with pytest.raises(mz.MzError) as e:
        mz.mz_q4_gemm(1, 10, 128, 64, 1, 0, 1)          # n_pad not a multiple of 256
    assert e.value.status == mz.MZ_EINVAL
    with pytest.raises(mz.MzError):
        mz.mz_attention(1, 1, 4, 1, 1, 1, 16, 6, 4, 64, 1)   # 6 q heads over 4 kv heads
    with pytest.raises(mz.MzError):
        mz.mz_attention(1, 1, 4, 1, 1, 8193, 16, 8, 2, 64, 1)   # a chunk table above 8192 entries
    with pytest.raises(mz.MzError):
        mz.mz_attention_split(1, 1, 4, 10, 1, 1, 8193, 16, 8, 2, 64, 2, 1, 1 << 30, 1)


@pytest.mark.parametrize("n,scale_kind", [(64, "normal"), (4096, "normal"), (64 * 1237, "mixed"),
                                          (524288, "normal"), (640, "special")])
def test_kv_codec_bit_exact(n, scale_kind):
    """Swap-path codec: codes, per-group (min, step) and reconstruction equal
    the oracle's bit for bit (same fp32 steps, correctly rounded division)."""
    from oracle import kv_codec as Q
    torch = torch_cuda()
    rng = np.random.default_rng(n)
    if scale_kind == "normal":
        x = (rng.standard_normal(n) * 1.7).astype(np.float16)
    elif scale_kind == "mixed":        # per-group scales from 1e-4 to 3e3, offsets
        g = n // 64
        x = (rng.standard_normal((g, 64)) * 10.0 ** rng.uniform(-4, 3.5, (g, 1))
             + rng.uniform(-100, 100, (g, 1))).astype(np.float16).reshape(-1)
    else:                              # constant, two-valued, subnormal, +-0, huge range, ties
        x = np.zeros(n, np.float16)
        x[64:128] = 2.5
        x[128:192] = np.where(np.arange(64) % 2, 1.0, -1.0)
        x[192:256] = np.float16(2.0 ** -20) * np.arange(64)
        x[256:320] = np.where(np.arange(64) % 3 == 0, -0.0, 0.0)
        x[320:384] = np.linspace(-60000, 60000, 64)
        x[384:448] = (np.arange(64) * 0.5 / 16).astype(np.float16)
        x[448:640] = rng.standard_normal(192)
    report("codec", n=n, kind=scale_kind)
    ref = Q.compress(x)
    d_x = torch.from_numpy(x.view(np.int16)).cuda()
    d_c = torch.empty(Q.compressed_bytes(n), dtype=torch.uint8, device="cuda")
    d_y = torch.empty(n, dtype=torch.int16, device="cuda")
    mz.mz_kv_compress(d_x.data_ptr(), n, d_c.data_ptr(), stream())
    mz.mz_kv_decompress(d_c.data_ptr(), n, d_y.data_ptr(), stream())
    torch.cuda.synchronize()
    got = d_c.cpu().numpy()
    assert np.array_equal(got[:n], ref[:n]), "codes"
    assert np.array_equal(got[n:], ref[n:]), "group parameters"
    assert np.array_equal(d_y.cpu().numpy().view(np.float16).view(np.uint16),
                          Q.decompress(ref, n).view(np.uint16)), "reconstruction"
