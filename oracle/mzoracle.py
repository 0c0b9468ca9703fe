"""CPU oracle for the evict / restore / recompute path behind time-to-first-token.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import this module.  The product path (the HIP engine and
its binding) never calls it, and this module shares no code with that path.

What it computes, and where each step comes from:

* The model is a stack of transformer layers whose prefill computes, for every
  token and every layer, a key and a value vector that are kept as the KV cache
  (paper, Sec. 2.1).  The layer is Llama-style (the paper does not fix it):
  RMSNorm (gain 1) -> Q/K/V projections -> rotary embedding on Q and K ->
  causal grouped-query attention -> output projection + residual -> RMSNorm ->
  SwiGLU feed-forward + residual; the first token is the argmax of the output
  head applied to the RMSNorm of the last position's final hidden state.
* Weights are Q4_0: a block of 32 weights shares one half-precision scale d
  and stores 4-bit codes q, the weight being d * (q - 8).
* The KV cache is split per layer into fixed-size token chunks and the weights
  into per-layer units (Sec. 4.2).  Each unit is resident, swapped to host
  memory, or dropped.  Eviction follows the caller's order, backward-out by
  default; restoration brings units back forward-in (Sec. 4.4).  A swapped unit
  comes back byte for byte.  A dropped KV chunk is recomputed (this is the
  re-targeting of the cold-start recompute, Sec. 1 and Sec. 3.1, to single
  chunks): a position p must pass through layer l whenever some layer l' >= l
  dropped the chunk holding p, so the rows of layer l are
      R_l = {p < N : chunk(p) dropped at some l' >= l} U {N..S-1} U {S-1}
  and the rows whose layer-l K/V is written are
      D_l = {p < N : chunk(p) dropped at layer l} U {N..S-1}.
* Attention of a query at position p reads every key j <= p of its layer from
  the chunked cache, whatever path restored each chunk (Sec. 4.2).

Precision: float64 everywhere except that K and V are stored as IEEE half
(round to nearest even) and read back from the stored halves, as the cache
format prescribes.

Parity pins (what ties this module to something other than itself) live in
tests/test_oracle_pins.py: brute-force attention, the Q4_0 closed form,
RMSNorm / RoPE / SiLU identities, causality and head-permutation structure,
and the two restore invariants (recomputed KV equals a clean prefill's; the
first-token logits after any plan equal the never-evicted logits).
"""

from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

RES, SWAP, DROP = 0, 1, 2


# ----------------------------------------------------------------------------- hyper-parameters

class Hyper:
    """Model shape read from any object (or dict) carrying the usual fields."""

    FIELDS = ("n_layers", "d_model", "n_q_heads", "n_kv_heads", "head_dim", "d_ffn", "vocab",
              "rope_theta", "rms_eps", "chunk_tokens")

    def __init__(self, src):
        get = (lambda k: src[k]) if isinstance(src, dict) else (lambda k: getattr(src, k))
        for k in self.FIELDS:
            setattr(self, k, get(k))
        self.n_layers = int(self.n_layers)
        self.dq = self.n_q_heads * self.head_dim
        self.dkv = self.n_kv_heads * self.head_dim
        self.group = self.n_q_heads // self.n_kv_heads


# ----------------------------------------------------------------------------- Q4_0

def q4_0_row_bytes(cols: int) -> int:
    return ((cols + 31) // 32) * 18


def q4_0_decode(raw: np.ndarray, rows: int, cols: int) -> np.ndarray:
    """Decode Q4_0 rows into float64 [rows, cols]: w = d * (q - 8).

    A block is 18 bytes: a little-endian IEEE half scale d, then 16 bytes whose
    low nibble is element j and high nibble element j + 16.
    """
    nb = (cols + 31) // 32
    blocks = np.asarray(raw, dtype=np.uint8).reshape(rows, nb, 18)
    d = blocks[:, :, 0:2].copy().view(np.float16)[:, :, 0].astype(np.float64)
    qs = blocks[:, :, 2:18]
    q = np.concatenate([qs & 0x0F, qs >> 4], axis=2).astype(np.float64)    # [rows, nb, 32]
    w = d[:, :, None] * (q - 8.0)
    return w.reshape(rows, nb * 32)[:, :cols]


class Weights:
    """Blob parser: per-layer Wq, Wk, Wv, Wo, W_gate, W_up, W_down, then E and W_lm."""

    LAYER_TENSORS = ("wq", "wk", "wv", "wo", "wg", "wu", "wd")

    def __init__(self, hp: Hyper, blob: np.ndarray, threads: int = 1):
        self.hp = hp
        self.threads = threads
        self.blob = np.asarray(blob, dtype=np.uint8).reshape(-1)
        d, dq, dkv, ff, V = hp.d_model, hp.dq, hp.dkv, hp.d_ffn, hp.vocab
        shapes = {"wq": (dq, d), "wk": (dkv, d), "wv": (dkv, d), "wo": (d, dq),
                  "wg": (ff, d), "wu": (ff, d), "wd": (d, ff)}
        self.index: Dict[Tuple[str, int], Tuple[int, int, int]] = {}
        off = 0
        for l in range(hp.n_layers):
            for name in self.LAYER_TENSORS:
                r, c = shapes[name]
                self.index[(name, l)] = (off, r, c)
                off += r * q4_0_row_bytes(c)
        for name in ("emb", "lm"):
            self.index[(name, -1)] = (off, V, d)
            off += V * q4_0_row_bytes(d)
        if off != self.blob.size:
            raise ValueError(f"blob has {self.blob.size} bytes, the shape needs {off}")
        self._cache: Dict[int, Dict[str, np.ndarray]] = {}

    def raw(self, name: str, layer: int = -1) -> np.ndarray:
        off, r, c = self.index[(name, layer)]
        return self.blob[off: off + r * q4_0_row_bytes(c)]

    def layer_unit_bytes(self, layer: int) -> bytes:
        """All Q4_0 bytes of one layer (the weight unit of Sec. 4.2)."""
        off0 = self.index[("wq", layer)][0]
        off1, r, c = self.index[("wd", layer)]
        return self.blob[off0: off1 + r * q4_0_row_bytes(c)].tobytes()

    def tensor(self, name: str, layer: int = -1) -> np.ndarray:
        """Decode a whole tensor (rows split over `threads` threads: each row
        decodes on its own)."""
        off, r, c = self.index[(name, layer)]
        raw = self.raw(name, layer).reshape(r, q4_0_row_bytes(c))
        if self.threads <= 1 or r < 2 * self.threads:
            return q4_0_decode(raw, r, c)
        out = np.empty((r, c), dtype=np.float64)
        step = (r + self.threads - 1) // self.threads

        def part(r0: int):
            r1 = min(r, r0 + step)
            out[r0:r1] = q4_0_decode(raw[r0:r1], r1 - r0, c)

        from concurrent.futures import ThreadPoolExecutor
        with ThreadPoolExecutor(self.threads) as ex:
            list(ex.map(part, range(0, r, step)))
        return out

    def layer(self, l: int) -> Dict[str, np.ndarray]:
        if l not in self._cache:
            self._cache = {l: {n: self.tensor(n, l) for n in self.LAYER_TENSORS}}
        return self._cache[l]

    def rows(self, name: str, idx: Sequence[int]) -> np.ndarray:
        """Decode only some rows of E or W_lm."""
        off, r, c = self.index[(name, -1)]
        rb = q4_0_row_bytes(c)
        raw = self.blob[off: off + r * rb].reshape(r, rb)[np.asarray(idx, dtype=np.int64)]
        return q4_0_decode(raw, len(idx), c)


# ----------------------------------------------------------------------------- layer pieces

def rmsnorm(h: np.ndarray, eps: float) -> np.ndarray:
    """h / sqrt(mean(h^2) + eps) along the last axis (gain 1)."""
    return h / np.sqrt(np.mean(h * h, axis=-1, keepdims=True) + eps)


def rope(x: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Rotate-half rotary embedding of x [n, heads, hd] at absolute positions pos [n].

    Pair (i, i + hd/2) is rotated by the angle pos * theta^(-2i/hd).
    """
    hd = x.shape[-1]
    half = hd // 2
    inv = theta ** (-(2.0 * np.arange(half, dtype=np.float64)) / hd)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv[None, :]          # [n, half]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def silu(z: np.ndarray) -> np.ndarray:
    return z / (1.0 + np.exp(-z))


def causal_gqa_attention(q: np.ndarray, qpos: np.ndarray, k: np.ndarray, v: np.ndarray,
                         block: int = 64, threads: int = 1) -> np.ndarray:
    """o[i, h] = sum_{j <= qpos[i]} softmax_j(q[i,h] . k[j,g(h)] / sqrt(hd)) v[j,g(h)].

    q [n, nq, hd] at absolute positions qpos [n]; k, v [S, nkv, hd] hold keys for
    positions 0..S-1; g(h) = h // (nq / nkv).  The softmax subtracts the row max.

    The query heads of one KV head share its keys, so they are taken together
    as the rows of one product with that head's keys (no copy of K/V per query
    head).  Queries are taken `block` at a time only to bound memory; with
    threads > 1 the independent (query block, KV head) pieces run on that many
    threads with a single-threaded BLAS each: the same steps, bit for bit what
    the serial loop gives under a single-threaded BLAS (a multi-threaded BLAS
    may add the products of one piece in another order, an fp64 rounding).
    """
    n, nq, hd = q.shape
    nkv = k.shape[1]
    group = nq // nkv
    qpos = np.asarray(qpos, dtype=np.int64)
    scale = 1.0 / math.sqrt(hd)
    kg = [np.ascontiguousarray(k[:, g]) for g in range(nkv)]       # [S, hd] per KV head
    vg = [np.ascontiguousarray(v[:, g]) for g in range(nkv)]
    out = np.empty((n, nq, hd), dtype=np.float64)

    def piece(b0: int, g: int):
        pb = qpos[b0:b0 + block]
        nb = pb.size
        last = int(pb.max()) + 1
        heads = slice(g * group, (g + 1) * group)
        rows = q[b0:b0 + nb, heads].reshape(nb * group, hd)          # (query, head) rows
        s = (rows @ kg[g][:last].T).reshape(nb, group, last)
        s *= scale
        lo = int(pb.min()) + 1                                      # keys below lo are seen by every query
        if lo < last:
            after = np.arange(lo, last)[None, :] > pb[:, None]       # key after its query
            s[:, :, lo:last][np.broadcast_to(after[:, None, :], (nb, group, last - lo))] = -np.inf
        s -= s.max(axis=-1, keepdims=True)
        np.exp(s, out=s)
        s /= s.sum(axis=-1, keepdims=True)
        out[b0:b0 + nb, heads] = (s.reshape(nb * group, last) @ vg[g][:last]).reshape(nb, group, hd)

    work = [(b0, g) for b0 in range(0, n, block) for g in range(nkv)]
    if threads <= 1 or len(work) == 1:
        for b0, g in work:
            piece(b0, g)
    else:
        from concurrent.futures import ThreadPoolExecutor
        from threadpoolctl import threadpool_limits
        with threadpool_limits(1), ThreadPoolExecutor(threads) as ex:
            list(ex.map(lambda bg: piece(*bg), work))
    return out


def argmax_first(logits: np.ndarray) -> int:
    """Greedy token: largest logit, lowest index on ties."""
    return int(np.argmax(logits))


def f16(x: np.ndarray) -> np.ndarray:
    return np.asarray(x, dtype=np.float64).astype(np.float16)


def layer_forward(hp: Hyper, w: Dict[str, np.ndarray], h: np.ndarray, pos: np.ndarray,
                  kv_write, kv_read, threads: int = 1, mlp_rows: int = 8192) -> np.ndarray:
    """One decoder layer over the rows h [n, d] at positions pos.

    kv_write(k_f16 [n, dkv], v_f16 [n, dkv]) stores the rows' keys/values
    wherever the caller decides; kv_read(last) returns (K, V) float64 [last, dkv]
    for positions 0..last-1 as stored.  The feed-forward block acts on each row
    alone; it runs mlp_rows rows at a time only to bound memory.
    """
    n = h.shape[0]
    x = rmsnorm(h, hp.rms_eps)
    q = (x @ w["wq"].T).reshape(n, hp.n_q_heads, hp.head_dim)
    k = (x @ w["wk"].T).reshape(n, hp.n_kv_heads, hp.head_dim)
    v = (x @ w["wv"].T).reshape(n, hp.n_kv_heads, hp.head_dim)
    del x
    q = rope(q, pos, hp.rope_theta)
    k = rope(k, pos, hp.rope_theta)
    kv_write(f16(k.reshape(n, hp.dkv)), f16(v.reshape(n, hp.dkv)))
    del k, v
    last = int(np.max(pos)) + 1
    K, V = kv_read(last)
    o = causal_gqa_attention(q, pos, K.reshape(last, hp.n_kv_heads, hp.head_dim),
                             V.reshape(last, hp.n_kv_heads, hp.head_dim), threads=threads)
    del q, K, V
    h = h + o.reshape(n, hp.dq) @ w["wo"].T
    del o
    for r0 in range(0, n, mlp_rows):
        y = rmsnorm(h[r0:r0 + mlp_rows], hp.rms_eps)
        h[r0:r0 + mlp_rows] += (silu(y @ w["wg"].T) * (y @ w["wu"].T)) @ w["wd"].T
    return h


def output_logits(hp: Hyper, wts: Weights, h_last: np.ndarray, block: int = 16384) -> np.ndarray:
    """logits = RMSNorm(h_last) . W_lm^T (vocabulary rows decoded a slice at a time)."""
    x = rmsnorm(h_last.reshape(1, -1), hp.rms_eps)[0]
    out = np.empty(hp.vocab, np.float64)
    for v0 in range(0, hp.vocab, block):
        idx = np.arange(v0, min(hp.vocab, v0 + block))
        out[idx] = wts.rows("lm", idx) @ x
    return out


# ----------------------------------------------------------------------------- clean prefill

def clean_prefill(hp: Hyper, wts: Weights, tokens: np.ndarray, threads: int = 1, progress=None):
    """Never-evicted prefill of all tokens: per-layer fp16 K, V [S, dkv] and the logits."""
    tokens = np.asarray(tokens, dtype=np.int64)
    S = tokens.size
    pos = np.arange(S)
    h = wts.rows("emb", tokens)
    Ks, Vs = [], []
    for l in range(hp.n_layers):
        K = np.zeros((S, hp.dkv), np.float16)
        V = np.zeros((S, hp.dkv), np.float16)

        def write(k, v, K=K, V=V):
            K[:], V[:] = k, v

        def read(last, K=K, V=V):
            return K[:last].astype(np.float64), V[:last].astype(np.float64)

        h = layer_forward(hp, wts.layer(l), h, pos, write, read, threads=threads)
        Ks.append(K)
        Vs.append(V)
        if progress:
            progress(l)
    logits = output_logits(hp, wts, h[-1])
    return Ks, Vs, logits


# ----------------------------------------------------------------------------- the method

def restore_rows(kv_state: np.ndarray, n_ctx: int, n_prompt: int, chunk: int):
    """R_l and D_l (sorted position arrays) for every layer."""
    L = kv_state.shape[0]
    S = n_ctx + n_prompt
    ctx_pos = np.arange(n_ctx)
    ch = ctx_pos // chunk
    prompt = np.arange(n_ctx, S)
    R, D = [], []
    for l in range(L):
        needed = (kv_state[l:, :] == DROP).any(axis=0)          # dropped at some l' >= l
        r = set(ctx_pos[needed[ch]].tolist()) | set(prompt.tolist()) | {S - 1}
        dset = set(ctx_pos[kv_state[l, ch] == DROP].tolist()) | set(prompt.tolist())
        R.append(np.array(sorted(r), dtype=np.int64))
        D.append(np.array(sorted(dset), dtype=np.int64))
    return R, D


class OracleContext:
    """The evict / restore / first-token sequence, one step at a time.

    Mirrors the engine's calls: prefill_context or import_kv build the cached
    context; evict applies a plan (swap to a host store or drop, per unit);
    restore_and_prefill brings swapped units back byte for byte and recomputes
    dropped chunks over R_l / D_l; first_token returns (token, logits).
    """

    def __init__(self, hyper, blob: np.ndarray, threads: int = 1):
        self.hp = Hyper(hyper)
        self.threads = threads
        self.wts = Weights(self.hp, blob, threads=threads)
        L, C = self.hp.n_layers, self.hp.chunk_tokens
        self.C = C
        self.tokens = np.zeros(0, np.int64)
        # per layer, per chunk: (K [C, dkv] f16, V [C, dkv] f16) or None when not resident
        self.chunks: List[List[Optional[Tuple[np.ndarray, np.ndarray]]]] = [[] for _ in range(L)]
        self.kv_state = np.zeros((L, 0), np.uint8)
        self.w_state = np.zeros(L, np.uint8)
        self.w_dev: List[Optional[bytes]] = [self.wts.layer_unit_bytes(l) for l in range(L)]
        self.host_kv: Dict[Tuple[int, int], Tuple[np.ndarray, np.ndarray]] = {}
        self.host_w: Dict[int, bytes] = {}
        self.swap_log: List[Tuple[str, int, int]] = []       # push order of swapped units
        self.restore_log: List[Tuple[str, int, int]] = []    # pop order at restore
        self.h_last: Optional[np.ndarray] = None
        self.stats = {}

    # -- context building
    @property
    def n_ctx(self) -> int:
        return int(self.tokens.size)

    def _alloc_chunks(self, n_tokens: int):
        n = (n_tokens + self.C - 1) // self.C
        for l in range(self.hp.n_layers):
            while len(self.chunks[l]) < n:
                self.chunks[l].append((np.zeros((self.C, self.hp.dkv), np.float16),
                                       np.zeros((self.C, self.hp.dkv), np.float16)))
        if self.kv_state.shape[1] < n:
            pad = np.zeros((self.hp.n_layers, n - self.kv_state.shape[1]), np.uint8)
            self.kv_state = np.concatenate([self.kv_state, pad], axis=1)

    def prefill_context(self, tokens: np.ndarray):
        tokens = np.asarray(tokens, dtype=np.int64)
        Ks, Vs, logits = clean_prefill(self.hp, self.wts, tokens, threads=self.threads)
        self.tokens = tokens.copy()
        self.chunks = [[] for _ in range(self.hp.n_layers)]
        self.kv_state = np.zeros((self.hp.n_layers, 0), np.uint8)
        self._alloc_chunks(tokens.size)
        for l in range(self.hp.n_layers):
            for p0 in range(0, tokens.size, self.C):
                p1 = min(tokens.size, p0 + self.C)
                K, V = self.chunks[l][p0 // self.C]
                K[: p1 - p0], V[: p1 - p0] = Ks[l][p0:p1], Vs[l][p0:p1]
        return logits

    def set_context(self, tokens: np.ndarray):
        """Declare the context tokens (their KV arrives through import_kv)."""
        self.tokens = np.asarray(tokens, dtype=np.int64).copy()
        self.chunks = [[] for _ in range(self.hp.n_layers)]
        self.kv_state = np.zeros((self.hp.n_layers, 0), np.uint8)
        self._alloc_chunks(self.tokens.size)

    def import_kv(self, layer: int, chunk: int, K: np.ndarray, V: np.ndarray):
        self.chunks[layer][chunk] = (np.array(K, np.float16).reshape(self.C, self.hp.dkv).copy(),
                                     np.array(V, np.float16).reshape(self.C, self.hp.dkv).copy())

    def read_kv(self, layer: int, chunk: int):
        c = self.chunks[layer][chunk]
        if c is None:
            raise RuntimeError("chunk is not resident")
        return c[0].copy(), c[1].copy()

    # -- eviction (idle phase)
    def evict(self, kv_state: np.ndarray, w_state: Optional[np.ndarray] = None,
              order: Optional[Sequence[Tuple[str, int, int]]] = None, codec: bool = False):
        """Apply a plan.  Units are visited in `order` (default backward-out:
        last layer first; within a layer its KV chunks from the last, then its
        weight unit), each moving RES -> SWAP / DROP or SWAP -> DROP.  With
        codec, a swapped chunk holding chunk_tokens positions is kept in the
        8-bit swap codec's form (oracle/kv_codec.py) and comes back as its
        round trip; partial chunks are kept as they are."""
        L = self.hp.n_layers
        nc = self.kv_state.shape[1]
        kv_state = np.asarray(kv_state, dtype=np.uint8)
        if kv_state.shape != (L, nc):
            raise ValueError("plan shape does not match the cached context")
        w_state = np.zeros(L, np.uint8) if w_state is None else np.asarray(w_state, np.uint8)
        if order is None:
            order = []
            for l in range(L - 1, -1, -1):
                order += [("kv", l, c) for c in range(nc - 1, -1, -1)]
                order.append(("w", l, -1))
        for kind, l, c in order:
            if kind == "kv":
                tgt, cur = int(kv_state[l, c]), int(self.kv_state[l, c])
                if tgt == RES or tgt == cur:
                    continue
                if tgt == SWAP and cur == DROP:
                    raise RuntimeError("cannot swap a dropped chunk")
                if tgt == SWAP:
                    k, v = self.chunks[l][c][0].copy(), self.chunks[l][c][1].copy()
                    if codec and (c + 1) * self.C <= self.n_ctx:
                        from .kv_codec import roundtrip_chunk
                        k, v = roundtrip_chunk(k, v)
                    self.host_kv[(l, c)] = (k, v)
                    self.swap_log.append(("kv", l, c))
                else:
                    self.host_kv.pop((l, c), None)
                self.chunks[l][c] = None
                self.kv_state[l, c] = tgt
            else:
                tgt, cur = int(w_state[l]), int(self.w_state[l])
                if tgt == RES or tgt == cur:
                    continue
                if tgt == SWAP and cur == DROP:
                    raise RuntimeError("cannot swap a dropped weight unit")
                if tgt == SWAP:
                    self.host_w[l] = self.w_dev[l]
                    self.swap_log.append(("w", l, -1))
                else:
                    self.host_w.pop(l, None)
                self.w_dev[l] = None
                self.w_state[l] = tgt

    # -- inference phase
    def restore_and_prefill(self, prompt: np.ndarray, progress=None):
        hp, C = self.hp, self.C
        prompt = np.asarray(prompt, dtype=np.int64)
        N, P = self.n_ctx, prompt.size
        S = N + P
        if S == 0:
            raise RuntimeError("nothing to prefill")
        state = self.kv_state.copy()
        # 1. swapped units come back byte for byte, earliest layer first (forward-in)
        self.restore_log = []
        for l in range(hp.n_layers):
            if self.w_state[l] == SWAP:
                self.w_dev[l] = self.host_w.pop(l)
                self.restore_log.append(("w", l, -1))
            elif self.w_state[l] == DROP:
                self.w_dev[l] = self.wts.layer_unit_bytes(l)      # reload from the model image
            for c in range(state.shape[1]):
                if state[l, c] == SWAP:
                    K, V = self.host_kv.pop((l, c))
                    self.chunks[l][c] = (K, V)
                    self.restore_log.append(("kv", l, c))
                elif state[l, c] == DROP:
                    self.chunks[l][c] = (np.zeros((C, hp.dkv), np.float16),
                                         np.zeros((C, hp.dkv), np.float16))
        for l in range(hp.n_layers):
            if self.w_dev[l] != self.wts.layer_unit_bytes(l):
                raise AssertionError("restored weight unit differs from the model image")
        # 2. rows that must pass through each layer, and rows whose K/V is written
        R, D = restore_rows(state, N, P, C)
        self.stats = {"nR": [int(r.size) for r in R], "nD": [int(d.size) for d in D]}
        all_tokens = np.concatenate([self.tokens, prompt])
        self._alloc_chunks(S)
        # 3. layer by layer over R_l
        h = self.wts.rows("emb", all_tokens[R[0]])
        for l in range(hp.n_layers):
            pos = R[l]
            dmask = np.isin(pos, D[l])
            layer_chunks = self.chunks[l]

            def write(k, v, pos=pos, dmask=dmask, layer_chunks=layer_chunks):
                for i in np.nonzero(dmask)[0]:
                    p = int(pos[i])
                    Kc, Vc = layer_chunks[p // C]
                    Kc[p % C], Vc[p % C] = k[i], v[i]

            def read(last, layer_chunks=layer_chunks):
                nch = (last + C - 1) // C
                K = np.concatenate([layer_chunks[c][0] for c in range(nch)])[:last]
                V = np.concatenate([layer_chunks[c][1] for c in range(nch)])[:last]
                return K.astype(np.float64), V.astype(np.float64)

            h = layer_forward(hp, self.wts.layer(l), h, pos, write, read, threads=self.threads)
            if l + 1 < hp.n_layers:
                h = h[np.isin(pos, R[l + 1])]
            if progress:
                progress(l)
        self.h_last = h[-1].copy()           # R_l always ends with S-1
        self.tokens = all_tokens
        self.kv_state = np.zeros((hp.n_layers, (S + C - 1) // C), np.uint8)
        self.w_state[:] = RES
        return self.stats

    def first_token(self):
        if self.h_last is None:
            raise RuntimeError("restore_and_prefill has not run")
        logits = output_logits(self.hp, self.wts, self.h_last)
        return argmax_first(logits), logits
