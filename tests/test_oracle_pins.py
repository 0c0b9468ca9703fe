"""Pins for the CPU oracle: brute force, closed forms and invariants that do not
come from the oracle itself.  CPU only."""

import math
import os

import numpy as np
import pytest

import oracle as O
from paper_2609_01338_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ----------------------------------------------------------------------------- Q4_0

def _block(d_bits: int, nibbles_lo, nibbles_hi) -> bytes:
    qs = bytes((lo & 0xF) | ((hi & 0xF) << 4) for lo, hi in zip(nibbles_lo, nibbles_hi))
    return bytes([d_bits & 0xFF, d_bits >> 8]) + qs


def test_q4_0_closed_form_hand_block():
    # d = 0.5 (half 0x3800); element j < 16 has code j, element j+16 has code 15-j
    raw = np.frombuffer(_block(0x3800, range(16), [15 - j for j in range(16)]), np.uint8)
    w = O.q4_0_decode(raw, 1, 32)[0]
    expect = [0.5 * (j - 8) for j in range(16)] + [0.5 * (7 - j) for j in range(16)]
    assert w.tolist() == expect
    # d = -0.25 (half 0xB400), all codes 0 -> +2.0
    raw = np.frombuffer(_block(0xB400, [0] * 16, [0] * 16), np.uint8)
    assert O.q4_0_decode(raw, 1, 32)[0].tolist() == [2.0] * 32
    # smallest subnormal half scale 2^-24, code 15 -> 7 * 2^-24 exactly
    raw = np.frombuffer(_block(0x0001, [15] * 16, [8] * 16), np.uint8)
    w = O.q4_0_decode(raw, 1, 32)[0]
    assert w[:16].tolist() == [7 * 2.0 ** -24] * 16 and w[16:].tolist() == [0.0] * 16


def test_q4_0_two_rows_two_blocks_order():
    # row-major rows of consecutive blocks; columns past `cols` are cut
    b = [_block(0x3C00, [k] * 16, [k] * 16) for k in (9, 10, 11, 12)]   # d = 1
    raw = np.frombuffer(b"".join(b), np.uint8)
    w = O.q4_0_decode(raw, 2, 40)
    assert w.shape == (2, 40)
    assert (w[0, :32] == 1).all() and (w[0, 32:] == 2).all()
    assert (w[1, :32] == 3).all() and (w[1, 32:] == 4).all()


def test_q4_0_encode_round_trip_bound():
    rng = np.random.default_rng(3)
    x = (rng.standard_normal((64, 96)) * 0.02).astype(np.float32)
    x[5] = 0.0                                               # zero row -> scale 0, codes 8
    x[7, 40:] = 0.0
    raw = W.encode_q4_0(x)
    xh = O.q4_0_decode(raw.reshape(-1), 64, 96)
    assert (xh[5] == 0).all()
    blocks = raw.reshape(64, 3, 18)
    d = np.abs(blocks[:, :, :2].copy().view(np.float16)[:, :, 0].astype(np.float64))
    err = np.abs(x.astype(np.float64) - xh).reshape(64, 3, 32)
    amax = np.abs(x.astype(np.float64)).reshape(64, 3, 32).max(-1)
    # |x - x^| <= d/2, plus |q - 8| <= 8 times the half rounding of d (2^-11 relative);
    # only code 15 can be clamped (x/d in [7.5, 8] maps to 7d), with error at most about d
    qs = blocks[:, :, 2:]
    codes = np.concatenate([qs & 15, qs >> 4], axis=2)
    slack = np.broadcast_to(d[..., None] * 2.0 ** -7 + 1e-12, err.shape)
    half = np.broadcast_to(0.5 * d[..., None], err.shape)
    assert (err[codes < 15] <= (half + slack)[codes < 15]).all()
    assert (err <= d[..., None] + slack).all()
    # the largest-magnitude element reconstructs to -8 d_half ~ m
    i = np.abs(x[0, :32]).argmax()
    assert abs(xh[0, i] - x[0, i]) <= abs(x[0, i]) * 2.0 ** -10


def test_q4_0_padding_decodes_to_zero():
    rng = np.random.default_rng(4)
    x = rng.standard_normal((3, 40)).astype(np.float32)
    raw = W.encode_q4_0(x)                 # 2 blocks per row, second block half padding
    full = O.q4_0_decode(raw.reshape(-1), 3, 64)
    assert (full[:, 40:] == 0).all()


# ----------------------------------------------------------------------------- attention

def _brute_attention(q, qpos, k, v):
    n, nq, hd = q.shape
    nkv = k.shape[1]
    g = nq // nkv
    out = np.zeros_like(q)
    for i in range(n):
        for h in range(nq):
            kvh = h // g
            scores = []
            for j in range(int(qpos[i]) + 1):
                s = 0.0
                for t in range(hd):
                    s += float(q[i, h, t]) * float(k[j, kvh, t])
                scores.append(s / math.sqrt(hd))
            m = max(scores)
            e = [math.exp(s - m) for s in scores]
            z = sum(e)
            for t in range(hd):
                out[i, h, t] = sum(e[j] / z * float(v[j, kvh, t]) for j in range(len(e)))
    return out


@pytest.mark.parametrize("nq,nkv", [(4, 2), (6, 2), (3, 1), (4, 4)])
def test_attention_matches_brute_force(nq, nkv):
    rng = np.random.default_rng(nq * 10 + nkv)
    S, hd = 13, 8
    qpos = np.array([0, 2, 3, 7, 11, 12])                    # gappy absolute positions
    q = rng.standard_normal((qpos.size, nq, hd)) * 1.5
    k = rng.standard_normal((S, nkv, hd)) * 1.5
    v = rng.standard_normal((S, nkv, hd))
    got = O.causal_gqa_attention(q, qpos, k, v, block=4)
    assert np.allclose(got, _brute_attention(q, qpos, k, v), rtol=0, atol=1e-12)


def test_attention_special_cases():
    rng = np.random.default_rng(7)
    S, hd = 9, 16
    k = rng.standard_normal((S, 2, hd))
    v = rng.standard_normal((S, 2, hd))
    # a query at position 0 sees one key: output is that value exactly
    q = rng.standard_normal((1, 4, hd))
    o = O.causal_gqa_attention(q, np.array([0]), k, v)
    assert np.array_equal(o[0, :2], v[0, [0, 0]]) and np.array_equal(o[0, 2:], v[0, [1, 1]])
    # zero query: equal scores -> mean of the visible values
    q = np.zeros((2, 4, hd))
    o = O.causal_gqa_attention(q, np.array([4, 8]), k, v)
    assert np.allclose(o[0, 0], v[:5, 0].mean(0), atol=1e-14)
    assert np.allclose(o[1, 3], v[:9, 1].mean(0), atol=1e-14)
    # one overwhelming score selects that key's value
    q = np.zeros((1, 2, hd))
    kk = np.zeros((S, 1, hd))
    kk[3, 0, 0] = 1.0
    q[0, :, 0] = 4000.0
    o = O.causal_gqa_attention(q, np.array([8]), kk, v[:, :1])
    assert np.allclose(o[0, 1], v[3, 0], atol=1e-12)
    # keys after the query never contribute
    v2 = v.copy()
    v2[6:] = 1e6
    q = rng.standard_normal((1, 4, hd))
    assert np.array_equal(O.causal_gqa_attention(q, np.array([5]), k, v),
                          O.causal_gqa_attention(q, np.array([5]), k, v2))


# ----------------------------------------------------------------------------- norm / rope / silu

def test_rmsnorm_values():
    h = np.array([[3.0, 4.0]])
    assert np.allclose(O.rmsnorm(h, 0.0), [[3 / math.sqrt(12.5), 4 / math.sqrt(12.5)]], atol=1e-15)
    rng = np.random.default_rng(1)
    h = rng.standard_normal((5, 64)) * 3
    eps = 1e-5
    y = O.rmsnorm(h, eps)
    ms = (h * h).mean(-1)
    assert np.allclose(np.sqrt((y * y).mean(-1)), np.sqrt(ms / (ms + eps)), atol=1e-14)
    assert np.allclose(O.rmsnorm(7.0 * h, 0.0), O.rmsnorm(h, 0.0), atol=1e-14)


def test_rope_values_and_properties():
    # hd = 2: one pair, frequency theta^0 = 1, so the angle is the position itself
    x = np.array([[[1.0, 0.0]]])
    y = O.rope(x, np.array([1]), 1e4)
    assert np.allclose(y, [[[math.cos(1.0), math.sin(1.0)]]], atol=1e-15)
    # hd = 4: second pair (1, 3) rotates at theta^(-1/2)
    x = np.array([[[0.0, 1.0, 0.0, 0.0]]])
    a = 3 * 100.0 ** -0.5
    y = O.rope(x, np.array([3]), 100.0)
    assert np.allclose(y, [[[0.0, math.cos(a), 0.0, math.sin(a)]]], atol=1e-15)
    rng = np.random.default_rng(2)
    q = rng.standard_normal((1, 3, 16))
    k = rng.standard_normal((1, 3, 16))
    assert np.array_equal(O.rope(q, np.array([0]), 5e5), q)
    # per-pair norms preserved
    y = O.rope(q, np.array([1234]), 5e5)
    n0 = q[..., :8] ** 2 + q[..., 8:] ** 2
    n1 = y[..., :8] ** 2 + y[..., 8:] ** 2
    assert np.allclose(n0, n1, atol=1e-13)
    # q(m) . k(n) depends on m - n only
    def dot(m, n):
        return (O.rope(q, np.array([m]), 1e4) * O.rope(k, np.array([n]), 1e4)).sum(-1)
    assert np.allclose(dot(10, 3), dot(107, 100), atol=1e-12)
    assert np.allclose(dot(5, 5), (q * k).sum(-1), atol=1e-12)


def test_silu_values():
    assert O.silu(np.array([0.0]))[0] == 0.0
    z = np.array([-3.0, -0.5, 0.5, 2.0, 40.0])
    assert np.allclose(O.silu(z) - O.silu(-z), z, atol=1e-14)        # silu(z) - silu(-z) = z
    assert abs(O.silu(np.array([40.0]))[0] - 40.0) < 1e-15
    assert abs(O.silu(np.array([-40.0]))[0]) < 1e-15
    assert abs(O.silu(np.array([1.0]))[0] - 1.0 / (1.0 + math.exp(-1.0))) < 1e-16


def test_argmax_lowest_index_on_ties():
    assert O.argmax_first(np.array([1.0, 3.0, 3.0, 2.0])) == 1
    assert O.argmax_first(np.array([-1.0, -1.0])) == 0


# ----------------------------------------------------------------------------- model structure

TINY_HP = dict(n_layers=2, d_model=64, n_q_heads=4, n_kv_heads=2, head_dim=16, d_ffn=80,
               vocab=97, rope_theta=1e4, rms_eps=1e-5, chunk_tokens=8)


def _blob_from_floats(hp, tensors):
    """Encode float tensors given in blob order into a Q4_0 blob (input encoding)."""
    return np.concatenate([W.encode_q4_0(t).reshape(-1) for t in tensors])


def _random_tensors(hp, seed, scale=0.3):
    rng = np.random.default_rng(seed)
    d, dq, dkv, ff, V = (hp["d_model"], hp["n_q_heads"] * hp["head_dim"],
                         hp["n_kv_heads"] * hp["head_dim"], hp["d_ffn"], hp["vocab"])
    ts = []
    for _ in range(hp["n_layers"]):
        for r, c in ((dq, d), (dkv, d), (dkv, d), (d, dq), (ff, d), (ff, d), (d, ff)):
            ts.append((rng.standard_normal((r, c)) * scale / math.sqrt(c) * 4).astype(np.float32))
    ts.append(rng.standard_normal((V, d)).astype(np.float32))
    ts.append((rng.standard_normal((V, d)) * 0.2).astype(np.float32))
    return ts


def test_prefill_is_causal():
    hp = O.Hyper(TINY_HP)
    wts = O.Weights(hp, _blob_from_floats(TINY_HP, _random_tensors(TINY_HP, 0)))
    toks = np.random.default_rng(5).integers(0, hp.vocab, 30)
    K1, V1, _ = O.clean_prefill(hp, wts, toks[:21])
    K2, V2, _ = O.clean_prefill(hp, wts, toks)
    for l in range(hp.n_layers):
        assert np.array_equal(K1[l], K2[l][:21]) and np.array_equal(V1[l], V2[l][:21])


def test_zero_branches_give_embedding_logits():
    ts = _random_tensors(TINY_HP, 1)
    for l in range(TINY_HP["n_layers"]):
        ts[7 * l + 3][:] = 0.0        # Wo
        ts[7 * l + 6][:] = 0.0        # W_down
    hp = O.Hyper(TINY_HP)
    wts = O.Weights(hp, _blob_from_floats(TINY_HP, ts))
    toks = np.array([3, 50, 17, 96, 2])
    _, _, logits = O.clean_prefill(hp, wts, toks)
    e = O.q4_0_decode(W.encode_q4_0(ts[-2][[2]]).reshape(-1), 1, hp.d_model)[0]
    lm = O.q4_0_decode(W.encode_q4_0(ts[-1]).reshape(-1), hp.vocab, hp.d_model)
    x = e / math.sqrt((e * e).mean() + hp.rms_eps)
    assert np.allclose(logits, lm @ x, atol=1e-12)


def test_kv_head_permutation_invariance():
    hp = O.Hyper(TINY_HP)
    hd, G, nkv = hp.head_dim, hp.group, hp.n_kv_heads
    ts = _random_tensors(TINY_HP, 2)
    perm = [1, 0]                               # kv head g moves to perm[g]
    pt = [t.copy() for t in ts]
    for l in range(hp.n_layers):
        wq, wk, wv, wo = (ts[7 * l + i] for i in range(4))
        for g in range(nkv):
            ng = perm[g]
            pt[7 * l + 1][ng * hd:(ng + 1) * hd] = wk[g * hd:(g + 1) * hd]
            pt[7 * l + 2][ng * hd:(ng + 1) * hd] = wv[g * hd:(g + 1) * hd]
            for r in range(G):
                src, dst = g * G + r, ng * G + r
                pt[7 * l + 0][dst * hd:(dst + 1) * hd] = wq[src * hd:(src + 1) * hd]
                pt[7 * l + 3][:, dst * hd:(dst + 1) * hd] = wo[:, src * hd:(src + 1) * hd]
    toks = np.random.default_rng(9).integers(0, hp.vocab, 19)
    Ka, Va, la = O.clean_prefill(hp, O.Weights(hp, _blob_from_floats(TINY_HP, ts)), toks)
    Kb, Vb, lb = O.clean_prefill(hp, O.Weights(hp, _blob_from_floats(TINY_HP, pt)), toks)
    assert np.allclose(la, lb, atol=1e-10)
    for l in range(hp.n_layers):
        for g in range(nkv):
            ng = perm[g]
            assert np.array_equal(Ka[l][:, g * hd:(g + 1) * hd], Kb[l][:, ng * hd:(ng + 1) * hd])


def test_layer_forward_closed_form():
    """One decoder layer (Sec. 2.1, in the Llama-style reading) on a shape small
    enough to work out by hand: d = 4, one query and one KV head of width 2,
    d_ffn = 1, eps = 0, two rows at positions 0 and 1.  Every weight is 0 or 1,
    which Q4_0 represents exactly (scale 1, codes 8 and 9).

      Wq picks (x1, x2), Wk picks (x2, x1), Wv picks (x3, x4); Wo adds o to
      (h1, h2); W_gate picks y1, W_up picks y3, W_down adds to h4.

    With h0 = (1, 1, 1, 1) and h1 = (1, -1, 1, -1) both rows have RMS 1, so
    x = h.  At position 1 the single rotary pair turns by 1 radian
    (theta^0 = 1), so with c = cos 1, s = sin 1:
      q1 = (c + s, s - c), k1 = (-c - s, c - s), and q0 = k0 = v0 = (1, 1),
      v1 = (1, -1) (values are not rotated).
    Keys are stored in half precision and read back, so k1 enters the scores
    as half(k1).  Query 0 sees only key 0: o0 = v0.  Query 1 scores
      z0 = q1 . k0 / sqrt 2,  z1 = q1 . half(k1) / sqrt 2,
    a = softmax(z0, z1), o1 = a0 v0 + a1 v1.  Then h' = h + (o, 0, 0),
    y = h' / rms(h'), and h'' = h' + (0, 0, 0, silu(y1) * y3).

    A gate/up swap, a rotation of V, a missing rotation of K, the wrong score
    scale, the second norm taken before the attention residual, or a dropped
    residual each change these numbers."""
    hp = O.Hyper(dict(n_layers=1, d_model=4, n_q_heads=1, n_kv_heads=1, head_dim=2, d_ffn=1,
                      vocab=2, rope_theta=1e4, rms_eps=0.0, chunk_tokens=8))
    w = {"wq": np.array([[1, 0, 0, 0], [0, 1, 0, 0]], float),
         "wk": np.array([[0, 1, 0, 0], [1, 0, 0, 0]], float),
         "wv": np.array([[0, 0, 1, 0], [0, 0, 0, 1]], float),
         "wo": np.array([[1, 0], [0, 1], [0, 0], [0, 0]], float),
         "wg": np.array([[1, 0, 0, 0]], float),
         "wu": np.array([[0, 0, 1, 0]], float),
         "wd": np.array([[0], [0], [0], [1]], float)}
    for m in w.values():                                   # Q4_0-exact weights
        assert np.array_equal(O.q4_0_decode(W.encode_q4_0(m.astype(np.float32)).reshape(-1), *m.shape), m)
    h = np.array([[1.0, 1.0, 1.0, 1.0], [1.0, -1.0, 1.0, -1.0]])
    store = {}

    def write(k, v):
        store["k"], store["v"] = k.copy(), v.copy()

    def read(last):
        return store["k"][:last].astype(np.float64), store["v"][:last].astype(np.float64)

    out = O.layer_forward(hp, w, h, np.array([0, 1]), write, read)

    c, s = math.cos(1.0), math.sin(1.0)
    k1h = [float(np.float16(-c - s)), float(np.float16(c - s))]
    assert store["k"].tolist() == [[1.0, 1.0], k1h]
    assert store["v"].tolist() == [[1.0, 1.0], [1.0, -1.0]]
    q1 = (c + s, s - c)
    z0 = (q1[0] * 1.0 + q1[1] * 1.0) / math.sqrt(2.0)
    z1 = (q1[0] * k1h[0] + q1[1] * k1h[1]) / math.sqrt(2.0)
    e0, e1 = math.exp(z0 - max(z0, z1)), math.exp(z1 - max(z0, z1))
    a0, a1 = e0 / (e0 + e1), e1 / (e0 + e1)
    o = [(1.0, 1.0), (a0 + a1, a0 - a1)]

    def silu(z):
        return z / (1.0 + math.exp(-z))

    expect = []
    for r in range(2):
        hr = [h[r, 0] + o[r][0], h[r, 1] + o[r][1], h[r, 2], h[r, 3]]
        rms = math.sqrt(sum(t * t for t in hr) / 4.0)
        y1, y3 = hr[0] / rms, hr[2] / rms
        expect.append([hr[0], hr[1], hr[2], hr[3] + silu(y1) * y3])
    assert np.allclose(out, expect, rtol=0, atol=1e-14)
    # the hand numbers at a glance: row 0 is (2, 2, 1, 1 + silu(2/sqrt 2.5)/sqrt 2.5)
    assert abs(out[0, 3] - (1.0 + silu(2 / math.sqrt(2.5)) / math.sqrt(2.5))) < 1e-14


# ----------------------------------------------------------------------------- rows R_l / D_l

def _brute_rows(state, N, P, C):
    L = state.shape[0]
    S = N + P
    R, D = [], []
    for l in range(L):
        r, d = [], []
        for p in range(S):
            if p >= N:
                r.append(p)
                d.append(p)
                continue
            c = p // C
            if any(state[m, c] == O.DROP for m in range(l, L)) or p == S - 1:
                r.append(p)
            if state[l, c] == O.DROP:
                d.append(p)
        R.append(r)
        D.append(d)
    return R, D


def test_restore_rows_brute_force():
    rng = np.random.default_rng(0)
    for trial in range(20):
        L, nc, C = 3, 5, 4
        N = int(rng.integers(1, nc * C + 1))
        nc = (N + C - 1) // C
        P = int(rng.integers(0, 6))
        state = rng.integers(0, 3, (L, nc)).astype(np.uint8)
        R, D = O.restore_rows(state, N, P, C)
        bR, bD = _brute_rows(state, N, P, C)
        assert [r.tolist() for r in R] == bR and [d.tolist() for d in D] == bD
        for l in range(L - 1):
            assert set(R[l + 1].tolist()) <= set(R[l].tolist())
        for l in range(L):
            assert set(D[l].tolist()) <= set(R[l].tolist())


def test_restore_rows_special_plans():
    L, N, P, C = 4, 40, 3, 8
    R, D = O.restore_rows(np.zeros((L, 5), np.uint8), N, P, C)
    assert all(r.tolist() == [40, 41, 42] for r in R)
    R, D = O.restore_rows(np.zeros((L, 5), np.uint8), N, 0, C)
    assert all(r.tolist() == [39] for r in R) and all(d.size == 0 for d in D)
    R, D = O.restore_rows(np.full((L, 5), O.DROP, np.uint8), N, P, C)
    assert all(r.tolist() == list(range(43)) for r in R)


# ----------------------------------------------------------------------------- restore invariants

TINY_W = W.WORKLOADS["tiny"]


@pytest.fixture(scope="module")
def tiny_model():
    blob = W.make_blob(TINY_W)
    ctx, _ = W.make_tokens(TINY_W)
    prm = np.random.default_rng(11).integers(0, TINY_W.model.vocab, 19).astype(np.int32)
    clean = {}
    hp = O.Hyper(TINY_W.model)
    wts = O.Weights(hp, blob)
    for P in (0, 5, 19):
        clean[P] = O.clean_prefill(hp, wts, np.concatenate([ctx, prm[:P]]))
    return blob, ctx, prm, clean


def _plans():
    L, nc = TINY_W.model.n_layers, TINY_W.n_chunks
    plans = [("all-res", np.zeros((L, nc), np.uint8), None),
             ("all-drop", np.full((L, nc), O.DROP, np.uint8), None),
             ("all-swap", np.full((L, nc), O.SWAP, np.uint8), None),
             ("workload", W.make_plan(TINY_W).kv_state, None)]
    for l in range(L):
        for c in range(nc):
            s = np.zeros((L, nc), np.uint8)
            s[l, c] = O.DROP
            plans.append((f"drop-{l}-{c}", s, None))
    for seed in range(8):
        p = W.random_plan(L, nc, 0.3, 0.3, seed, w_swap=0.3, w_drop=0.3)
        plans.append((f"rand-{seed}", p.kv_state, p.w_state))
    units = W.backward_out_units(L, nc)
    for k in (1, 5, 8, 12):
        s = np.zeros((L, nc), np.uint8)
        for l, c in units[:k]:
            s[l, c] = O.DROP
        plans.append((f"bo-drop-{k}", s, None))
    return plans


@pytest.mark.parametrize("P", [0, 5, 19])
def test_restore_invariants_many_plans(tiny_model, P):
    blob, ctx, prm, clean = tiny_model
    Kc, Vc, lc = clean[P]
    C = TINY_W.model.chunk_tokens
    S = ctx.size + P
    for name, kv, ws in _plans():
        ox = O.OracleContext(TINY_W.model, blob)
        ox.set_context(ctx)
        for l in range(TINY_W.model.n_layers):
            for c in range(TINY_W.n_chunks):
                ox.import_kv(l, c, clean[0][0][l][c * C:(c + 1) * C], clean[0][1][l][c * C:(c + 1) * C])
        pre = {(l, c): ox.read_kv(l, c) for l in range(TINY_W.model.n_layers) for c in range(TINY_W.n_chunks)}
        ox.evict(kv, ws)
        ox.restore_and_prefill(prm[:P])
        tok, logits = ox.first_token()
        for l in range(TINY_W.model.n_layers):
            for c in range((S + C - 1) // C):
                K, V = ox.read_kv(l, c)
                n = min(C, S - c * C)
                # invariant 1: every chunk equals the clean prefill's, bit for bit
                assert np.array_equal(K[:n], Kc[l][c * C:c * C + n]), (name, l, c)
                assert np.array_equal(V[:n], Vc[l][c * C:c * C + n]), (name, l, c)
                if c < TINY_W.n_chunks and kv[l, c] == O.SWAP:
                    assert K.tobytes() == pre[(l, c)][0].tobytes()
        # invariant 2: first-token logits equal the never-evicted ones
        assert np.allclose(logits, lc, rtol=0, atol=1e-9), name
        assert tok == O.argmax_first(lc)


def test_double_evict_and_order(tiny_model):
    blob, ctx, prm, clean = tiny_model
    L, nc = TINY_W.model.n_layers, TINY_W.n_chunks
    ox = O.OracleContext(TINY_W.model, blob)
    ox.prefill_context(ctx)
    s1 = np.full((L, nc), O.SWAP, np.uint8)
    ox.evict(s1, np.array([O.SWAP, O.RES], np.uint8))
    # backward-out pushes: last layer's chunks from the last, then its weight unit
    assert ox.swap_log[:nc] == [("kv", 1, c) for c in range(nc - 1, -1, -1)]
    assert ox.swap_log[nc + 0] == ("kv", 0, nc - 1) and ("w", 0, -1) in ox.swap_log
    s2 = np.zeros((L, nc), np.uint8)
    s2[1, 2:5] = O.DROP
    ox.evict(s2)
    with pytest.raises(RuntimeError):
        ox.evict(np.where(s2 == O.DROP, O.SWAP, O.RES).astype(np.uint8))
    ox.restore_and_prefill(prm[:5])
    # forward-in: restore pops from the earliest layer
    assert ox.restore_log[0] == ("w", 0, -1) and ox.restore_log[1] == ("kv", 0, 0)
    tok, logits = ox.first_token()
    assert np.allclose(logits, clean[5][2], atol=1e-9)


def test_partial_last_chunk(tiny_model):
    blob, ctx, prm, _ = tiny_model
    hp = O.Hyper(TINY_W.model)
    N = 117
    toks = np.concatenate([ctx[:N], prm[:7]])
    Kc, Vc, lc = O.clean_prefill(hp, O.Weights(hp, blob), toks)
    ox = O.OracleContext(TINY_W.model, blob)
    ox.prefill_context(ctx[:N])
    nc = (N + 15) // 16
    s = np.zeros((hp.n_layers, nc), np.uint8)
    s[0, nc - 1] = O.DROP
    s[1, 3] = O.SWAP
    ox.evict(s)
    ox.restore_and_prefill(prm[:7])
    tok, logits = ox.first_token()
    assert np.allclose(logits, lc, atol=1e-9)
    K, V = ox.read_kv(1, 7)
    assert np.array_equal(K[:124 - 112], Kc[1][112:124])


# ----------------------------------------------------------------------------- paper's worked numbers

def _golden(name):
    vals = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                k, v = line.split("=")
                vals[k.strip()] = float(v)
    return vals


def test_chunk_bytes_match_paper():
    g = _golden("chunk_accounting.txt")
    hp = O.Hyper(dict(n_layers=1, d_model=64, n_q_heads=4, n_kv_heads=4, head_dim=128, d_ffn=64,
                      vocab=8, rope_theta=1e4, rms_eps=1e-5, chunk_tokens=int(g["chunk_tokens"])))
    assert hp.dkv == g["kv_hidden"]
    blob = np.zeros(sum(r * ((c + 31) // 32) * 18 for r, c in
                        ((512, 64), (512, 64), (512, 64), (64, 512), (64, 64), (64, 64), (64, 64),
                         (8, 64), (8, 64))), np.uint8)
    ox = O.OracleContext(hp, blob)
    ox.set_context(np.zeros(int(g["context_tokens"]), np.int64))
    K, V = ox.read_kv(0, 0)
    assert K.nbytes + V.nbytes == g["chunk_bytes"]
    assert len(ox.chunks[0]) == g["context_tokens"] / g["chunk_tokens"]
    # an 8B-class KV cache at 32K context: 32 layers x 32768 x 1024 x 2 (K,V) x 2 bytes
    m = W.M8B
    assert m.n_layers * 32768 * m.dkv * 2 * 2 == g["kv_bytes_8b_32k"]


# ----------------------------------------------------------------------------- f16 operand floor

def test_f16_floor_reduces_to_fp64_oracle():
    """With the half-precision operand roundings switched off, the floor's
    prefill is the oracle's clean prefill bit for bit; with them on, it moves
    the keys and values (so the rounding is really applied) but stays within
    a few half ulps at this depth."""
    from oracle.f16_floor import f16_operand_floor, prefix_kv
    hp = O.Hyper(TINY_W.model)
    wts = O.Weights(hp, W.make_blob(TINY_W))
    ctx, _ = W.make_tokens(TINY_W)
    toks = ctx[:40]
    K0, V0, h0 = prefix_kv(hp, wts, toks, False)
    Kc, Vc, lc = O.clean_prefill(hp, wts, toks)
    for l in range(hp.n_layers):
        assert np.array_equal(K0[l], Kc[l].astype(np.float64))
        assert np.array_equal(V0[l], Vc[l].astype(np.float64))
    assert np.allclose(O.output_logits(hp, wts, h0), lc, rtol=0, atol=0)
    fl = f16_operand_floor(hp, wts, toks)
    kmax = max(np.abs(K0[l]).max() for l in range(hp.n_layers))
    assert fl.shape == (hp.n_layers,) and fl.max() > 0
    assert fl.max() <= 8 * 2.0 ** -11 * max(1.0, kmax)


def test_bf16_rounding_and_rounded_probability_attention():
    """The floor's bf16 rounding is round-to-nearest-even to 8 significant
    bits: hand values at the ties, and torch's own float32 -> bfloat16
    conversion on random values.  Its attention with rounded probabilities
    reduces to the oracle's attention when nothing is rounded."""
    from oracle.f16_floor import _attention_rounded_probs, _bf16
    t = [1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, 1.0 + 2.0 ** -8 + 2.0 ** -20, -(2.0 + 2.0 ** -7), 0.0]
    assert _bf16(np.array(t)).tolist() == [1.0, 1.0 + 2.0 ** -6, 1.0 + 2.0 ** -7, -2.0, 0.0]
    import torch
    x = np.random.default_rng(3).standard_normal(10000) * 10.0 ** np.random.default_rng(4).uniform(-6, 6, 10000)
    ref = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(_bf16(x.astype(np.float32)), ref)
    rng = np.random.default_rng(6)
    q = rng.standard_normal((7, 4, 8))
    k = rng.standard_normal((12, 2, 8))
    v = rng.standard_normal((12, 2, 8))
    pos = np.array([0, 1, 3, 5, 8, 10, 11])
    assert np.allclose(_attention_rounded_probs(q, pos, k, v, lambda a: a),
                       O.causal_gqa_attention(q, pos, k, v), rtol=0, atol=1e-13)


# ----------------------------------------------------------------------------- KV codec

def test_kv_codec_exact_grid_group():
    """A group lying on the grid m + j/16 with range 255/16: step, minimum
    and codes are known in closed form and the round trip is exact."""
    from oracle import kv_codec as Q
    codes = np.array(list(range(0, 252, 4)) + [255], np.int64)          # 64 codes, max 255
    x = (-8.0 + codes / 16.0).astype(np.float16)
    b = Q.compress(x)
    assert b.size == Q.compressed_bytes(64) == 68
    assert b[:64].tolist() == codes.tolist()
    m, d = b[64:].view(np.float16).tolist()
    assert m == -8.0 and d == 0.0625
    assert np.array_equal(Q.decompress(b, 64), x)


def test_kv_codec_special_groups():
    from oracle import kv_codec as Q
    const = np.full(64, 3.25, np.float16)                    # zero range: step 0, codes 0
    b = Q.compress(const)
    assert not b[:64].any() and b[64:].view(np.float16).tolist() == [3.25, 0.0]
    assert np.array_equal(Q.decompress(b, 64), const)
    # ties round to even: x - m = 0.5 d -> 0, 1.5 d -> 2 (d = 1/16, range 255/16)
    x = np.zeros(64, np.float16)
    x[1], x[2], x[3] = 0.5 / 16, 1.5 / 16, 255 / 16
    q = Q.compress(x)[:64]
    assert q[0] == 0 and q[1] == 0 and q[2] == 2 and q[3] == 255


def test_kv_codec_error_bound_and_no_accumulation():
    """|x^ - x| <= d/2 + half an ulp of x^ per element (one rounding to the
    grid, one to half precision); further swap cycles stay within that bound
    of the original (the codec does not accumulate error)."""
    from oracle import kv_codec as Q
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(64 * 2048) * np.repeat(rng.uniform(0.01, 30, 2048), 64)).astype(np.float16)
    b = Q.compress(x)
    d = np.repeat(b[x.size:].view(np.float16).reshape(-1, 2)[:, 1].astype(np.float64), 64)
    cur = x
    for cycle in range(4):
        cur = Q.decompress(Q.compress(cur), x.size)
        ulp = np.spacing(np.abs(cur).astype(np.float16)).astype(np.float64)
        err = np.abs(cur.astype(np.float64) - x.astype(np.float64))
        assert np.all(err <= 0.5 * d + 0.5 * ulp + 1e-12), cycle


def test_kv_codec_idempotent():
    """Repeated compression and decompression does not accumulate error (Sec.
    6).  On zero-centred groups of KV-like values (many scales), a value that
    has been through the codec once comes back from a second cycle as the same
    codes, the same (m, d) and the same halves, bit for bit.  A group far off
    zero relative to its range can move once more: the half rounding of its
    decoded maximum can shift the range by one ulp and so d by one half ulp;
    from the second cycle on it is a fixed point."""
    from oracle import kv_codec as Q
    rng = np.random.default_rng(5)
    n_groups = 4096
    scale = np.repeat(rng.uniform(1e-3, 40.0, n_groups), 64)
    x = (rng.standard_normal(64 * n_groups) * scale).astype(np.float16)
    x[:64] = 1.5                                            # constant group
    x[64:128] = np.where(rng.random(64) < 0.5, -2.0, 7.0)   # two-valued group
    b1 = Q.compress(x)
    y1 = Q.decompress(b1, x.size)
    b2 = Q.compress(y1)
    assert np.array_equal(b2, b1)
    assert Q.decompress(b2, x.size).tobytes() == y1.tobytes()
    # off-centre groups: a fixed point after the second cycle
    offset = np.repeat(rng.uniform(-60.0, 60.0, n_groups), 64)
    x = (rng.standard_normal(64 * n_groups) * scale + offset).astype(np.float16)
    y1 = Q.decompress(Q.compress(x), x.size)
    b2 = Q.compress(y1)
    y2 = Q.decompress(b2, x.size)
    assert np.array_equal(Q.compress(y2), b2)
    moved = (y1.reshape(-1, 64) != y2.reshape(-1, 64)).any(axis=1)
    assert moved.sum() <= n_groups // 1000


def test_kv_codec_chunk_order_round_trip():
    from oracle import kv_codec as Q
    rng = np.random.default_rng(1)
    k = rng.standard_normal((16, 128)).astype(np.float16)
    v = rng.standard_normal((16, 128)).astype(np.float16)
    flat = Q.chunk_device_order(k, v)
    assert np.array_equal(flat[16 * 128 + 5], v[5, 0]) and np.array_equal(flat[16 * 128 + 16], v[0, 1])
    k2, v2 = Q.chunk_from_device_order(flat, 16, 128)
    assert np.array_equal(k2, k) and np.array_equal(v2, v)
