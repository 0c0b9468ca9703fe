"""Host-side checks of the C ABI (no GPU needed): the library loads and
exports every function include/mz.h declares; the restore planner's rows
match the oracle's; the GEMM repacker lays Q4_0 blocks out as documented;
calls that need a device fail cleanly without one."""

import ctypes
import os
import re

import numpy as np
import pytest

import oracle as O
from paper_2609_01338_amd import mz
from paper_2609_01338_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module", autouse=True)
def built():
    if not os.path.exists(mz.LIB_PATH):
        from paper_2609_01338_amd import build
        build.build_all()
    mz.lib()


def _declared_functions():
    src = open(os.path.join(ROOT, "include", "mz.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(mz_[a-z0-9_]+)\s*\(", src)))


def test_exports_every_declared_symbol():
    names = _declared_functions()
    assert len(names) >= 19
    lib = ctypes.CDLL(mz.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert mz.mz_version().startswith("mz-mi355x")


def test_plan_rows_match_oracle():
    rng = np.random.default_rng(1)
    for trial in range(25):
        L = int(rng.integers(1, 5))
        C = int(rng.choice([4, 16, 256]))
        N = int(rng.integers(1, 6 * C))
        P = int(rng.integers(0, 2 * C))
        nc = (N + C - 1) // C
        st = rng.integers(0, 3, (L, nc)).astype(np.uint8)
        model = W.ModelConfig("t", L, 128, 2, 1, 64, 64, 32, 1e4, C)
        cfg = mz.make_cfg(model, N + P)
        nR, nD, R = mz.mz_plan_rows(cfg, st, N, P)
        oR, oD = O.restore_rows(st, N, P, C)
        assert nR.tolist() == [r.size for r in oR]
        assert nD.tolist() == [d.size for d in oD]
        for l in range(L):
            assert np.array_equal(R[l], oR[l])


def test_plan_rows_workloads():
    """Row counts of the five measured workloads (the sizes the bench times)."""
    for key in W.ORDERED_KEYS:
        w = W.WORKLOADS[key]
        plan = W.make_plan(w)
        cfg = mz.make_cfg(w.model, w.n_ctx + w.n_prompt)
        nR, nD, _ = mz.mz_plan_rows(cfg, plan.kv_state, w.n_ctx, w.n_prompt, with_rows=False)
        oR, oD = O.restore_rows(plan.kv_state, w.n_ctx, w.n_prompt, w.model.chunk_tokens)
        assert nR.tolist() == [r.size for r in oR], key
        assert nD.tolist() == [d.size for d in oD], key
    w = W.WORKLOADS["8b"]
    nR, nD, _ = mz.mz_plan_rows(mz.make_cfg(w.model, 32896), W.make_plan(w).kv_state, 32768, 128,
                                with_rows=False)
    assert nR[0] == 32896 and nD[0] == 128          # layers 0-7 resident: only the prompt is written


def test_plan_rows_errors():
    model = W.ModelConfig("t", 2, 128, 2, 1, 64, 64, 32, 1e4, 16)
    cfg = mz.make_cfg(model, 64)
    mz.mz_plan_rows(cfg, np.zeros((2, 3), np.uint8), 40, 0)        # 40 tokens need 3 chunks
    with pytest.raises(mz.MzError) as e:
        mz.mz_plan_rows(cfg, np.zeros((2, 2), np.uint8), 40, 0)
    assert e.value.status == mz.MZ_EINVAL
    with pytest.raises(mz.MzError):
        mz.mz_plan_rows(cfg, np.full((2, 3), 7, np.uint8), 40, 0)


def test_plan_rows_ok_case():
    model = W.ModelConfig("t", 2, 128, 2, 1, 64, 64, 32, 1e4, 16)
    cfg = mz.make_cfg(model, 64)
    st = np.zeros((2, 3), np.uint8)
    st[1, 1] = mz.MZ_DROP
    nR, nD, R = mz.mz_plan_rows(cfg, st, 40, 2)
    assert R[0].tolist() == list(range(16, 32)) + [40, 41]
    assert R[1].tolist() == list(range(16, 32)) + [40, 41]
    assert nD.tolist() == [2, 18]


def _codes_from_packed(nib16: np.ndarray) -> list:
    """The 32 codes of one packed block: dword i holds elements 8i..8i+7, element
    8i+2m at bits 4m and element 8i+2m+1 at bits 16+4m."""
    words = np.frombuffer(bytes(nib16), "<u4")
    out = [0] * 32
    for i in range(4):
        for m in range(4):
            out[8 * i + 2 * m] = int(words[i] >> (4 * m)) & 15
            out[8 * i + 2 * m + 1] = int(words[i] >> (16 + 4 * m)) & 15
    return out


def _codes_from_blob(block18: np.ndarray) -> list:
    qs = bytes(block18[2:])
    return [qs[j] & 15 for j in range(16)] + [qs[j] >> 4 for j in range(16)]


def test_gemm_pack_layout():
    """Tile (nt, kt) holds rows nt*256.., blocks kt*2..: code blocks (row, block) x 16 B,
    then the fp16 scales; padding rows/blocks carry scale 0."""
    rng = np.random.default_rng(2)
    n, k = 300, 96                       # n pads to 512, k to 128
    x = rng.standard_normal((n, k)).astype(np.float32)
    raw = W.encode_q4_0(x)               # [n, 3 blocks * 18]
    packed = mz.mz_q4_gemm_pack(raw, n, k)
    tiles = packed.reshape(2, 2, 9216)   # [n tiles][k tiles][bytes]
    blocks = raw.reshape(n, 3, 18)
    for nt in range(2):
        for kt in range(2):
            t = tiles[nt, kt]
            nib = t[:8192].reshape(256, 2, 16)
            sc = t[8192:].reshape(256, 2, 2)
            for r in (0, 5, 43, 44, 71, 255):
                row = nt * 256 + r
                for b in range(2):
                    blk = kt * 2 + b
                    if row < n and blk < 3:
                        assert _codes_from_packed(nib[r, b]) == _codes_from_blob(blocks[row, blk])
                        assert bytes(sc[r, b]) == bytes(blocks[row, blk, :2])
                    else:
                        assert bytes(sc[r, b]) == b"\0\0"


def test_gemm_pack_gateup_interleave():
    rng = np.random.default_rng(3)
    n, k = 40, 64                        # n pads to 128 per matrix -> 256 packed rows
    g = W.encode_q4_0(rng.standard_normal((n, k)).astype(np.float32))
    u = W.encode_q4_0(rng.standard_normal((n, k)).astype(np.float32))
    packed = mz.mz_q4_gemm_pack(g, n, k, w_up=u)
    assert packed.size == mz.mz_q4_gemm_packed_bytes(256, 64)
    nib = packed[:8192].reshape(256, 2, 16)
    gb, ub = g.reshape(n, 2, 18), u.reshape(n, 2, 18)
    for pr in range(256):
        grp, i = divmod(pr, 32)
        src = grp * 16 + (i if i < 16 else i - 16)
        if src < n:
            ref = (gb if i < 16 else ub)[src]
            assert _codes_from_packed(nib[pr, 1]) == _codes_from_blob(ref[1])


def test_load_model_without_gpu_fails_cleanly():
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    w = W.WORKLOADS["tiny"]
    blob = W.make_blob(w)
    with pytest.raises(mz.MzError) as e:
        mz.mz_load_model(mz.make_cfg(w.model, 256), blob, 0)
    assert e.value.status in (mz.MZ_EHIP, mz.MZ_EINVAL)
    # wrong blob size is rejected before any device call
    with pytest.raises(mz.MzError) as e:
        mz.mz_load_model(mz.make_cfg(w.model, 256), blob[:-1], 0)
    assert e.value.status == mz.MZ_EINVAL


def test_attention_auto_splits_decode_rows():
    """Split counts are host logic: for a decode row (the few-column kernel,
    one workgroup per key split and KV head) the count depends on the KV
    heads and the key range only, not on how many query heads share a KV
    head (which changes the tiled kernel's waves per workgroup); the 8B
    decode step over 32900 keys takes about one workgroup per CU."""
    counts = {g: mz.mz_attention_auto_splits(1, 16399, 2 * g, 2, 128, 64 << 20) for g in (1, 2, 3, 4, 6, 7)}
    assert len(set(counts.values())) == 1, counts
    assert 24 <= mz.mz_attention_auto_splits(1, 32899, 32, 8, 128, 64 << 20) <= 32
    assert mz.mz_attention_auto_splits(1, 32899, 24, 8, 128, 64 << 20) == \
        mz.mz_attention_auto_splits(1, 32899, 32, 8, 128, 64 << 20)
    assert mz.mz_attention_auto_splits(40000, 40000, 24, 8, 128, 64 << 20) == 1   # the chip is full already


def test_gemm_long_k_splits():
    """256-row tiles split over K only where they alone are too few for the
    chip, the 64-row tiles fill it, every split keeps 16 K steps and the
    partials fit the workspace: the 1B down projection (2048 rows, 2048
    outputs, K 8192) with the restore's 64 MiB takes 4 splits of 32 steps;
    its output projection (K 2048, 8 steps a split) and the 8B full-row
    products stay whole, few rows are left to the split-K rule for few
    rows."""
    ws = 64 << 20
    assert mz.mz_q4_gemm_long_k_splits(2048, 2048, 8192, ws) == 4
    assert mz.mz_q4_gemm_long_k_splits(2048, 2048, 8192, ws - 1) == 1      # partials would not fit
    assert mz.mz_q4_gemm_long_k_splits(2048, 2048, 4096, ws) == 4
    assert mz.mz_q4_gemm_long_k_splits(2048, 2048, 2048, ws) == 1
    assert mz.mz_q4_gemm_long_k_splits(32896, 4096, 14336, ws) == 1
    assert mz.mz_q4_gemm_long_k_splits(1024, 2048, 8192, ws) == 1          # 128 64-row tiles
    assert mz.mz_q4_gemm_long_k_splits(1536, 4096, 14336, 80 << 20) == 3
    assert mz.mz_q4_gemm_long_k_splits(1536, 4096, 14336, ws) == 1


def test_gemm_auto_splits_medium_rows():
    """Few rows split over K; from 1024 rows on, 64-row tiles that cover half
    the chip run whole (the 1B and 1.5B K/V projections); the rows after the
    last whole 256-row tile of a long product keep their split."""
    ws = 64 << 20
    assert mz.mz_q4_gemm_auto_splits(2048, 1024, 2048, ws) == 1
    assert mz.mz_q4_gemm_auto_splits(4979, 512, 1536, ws) == 1
    assert mz.mz_q4_gemm_auto_splits(1023, 2048, 2048, ws) > 1          # 128 tiles, fewer rows
    assert mz.mz_q4_gemm_auto_splits(1024, 2048, 2048, ws) == 1
    assert mz.mz_q4_gemm_auto_splits(128, 28672, 4096, ws) == 3
    assert mz.mz_q4_gemm_auto_splits(129, 4096, 4096, ws) > 1
