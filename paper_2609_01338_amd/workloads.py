"""Synthetic workloads for the evict / restore / recompute path.

This module only *generates inputs*: model shapes, seeded Q4_0 weight blobs,
context and prompt token ids, and eviction plans.  It holds no step of the
method (no dequantization, attention or model arithmetic); the CPU oracle and
the HIP engine each implement those on their own and both read what this
module writes.

Model: a Llama-style decoder with the five shapes used for measurement (tiny,
1B-, 3B-, 1.5B- and 8B-class).  Weights are drawn N(0, 0.02^2) and stored as
Q4_0; RMSNorm gains are 1 and are not stored.

Blob layout (the model file handed to ``mz_load_model``): for each layer
``l = 0..L-1`` the tensors Wq [dq, d], Wk [dkv, d], Wv [dkv, d], Wo [d, dq],
W_gate [ff, d], W_up [ff, d], W_down [d, ff]; then the embedding E [V, d] and
the output head W_lm [V, d].  Every tensor is ``[out][in]`` (y = x W^T) and is
stored row by row as ``ceil(in/32)`` Q4_0 blocks of 18 bytes (fp16 scale, then
16 bytes: element j in the low nibble of byte j, element j+16 in its high
nibble).  A row whose ``in`` is not a multiple of 32 is zero-padded, which
encodes to scale 0.

Eviction plans: ``kv_state[l, c]`` and ``w_state[l]`` take RES (0), SWAP (1) or
DROP (2), following the per-layer weight units and per-layer KV chunks of the
paper's fine-grained memory management (Sec. 4.2) and its backward-out order
(Sec. 4.4).
"""

from __future__ import annotations

import ctypes
import dataclasses
import os
import subprocess
from typing import List, Optional, Tuple

import numpy as np

RES, SWAP, DROP = 0, 1, 2

_HERE = os.path.dirname(os.path.abspath(__file__))
_SYNTH_SRC = os.path.join(_HERE, "synth", "synth.c")
_SYNTH_LIB = os.path.join(_HERE, "synth", "libmzsynth.so")


@dataclasses.dataclass(frozen=True)
class ModelConfig:
    name: str
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    d_ffn: int
    vocab: int
    rope_theta: float
    chunk_tokens: int
    rms_eps: float = 1e-5

    @property
    def dq(self) -> int:
        return self.n_q_heads * self.head_dim

    @property
    def dkv(self) -> int:
        return self.n_kv_heads * self.head_dim

    def with_layers(self, n_layers: int) -> "ModelConfig":
        return dataclasses.replace(self, n_layers=n_layers, name=f"{self.name}-L{n_layers}")


@dataclasses.dataclass(frozen=True)
class Workload:
    key: str
    config_id: int          # seeds the weight draws
    model: ModelConfig
    n_ctx: int              # tokens of cached context (N)
    n_prompt: int           # new prompt tokens (P)
    plan_rule: str          # how the eviction plan is drawn, see make_plan()
    description: str

    @property
    def n_chunks(self) -> int:
        c = self.model.chunk_tokens
        return (self.n_ctx + c - 1) // c

    def scaled(self, n_layers: Optional[int] = None, n_ctx: Optional[int] = None,
               n_prompt: Optional[int] = None) -> "Workload":
        """Same layer shape, fewer layers / shorter context (parity-test sizes)."""
        m = self.model if n_layers is None else self.model.with_layers(n_layers)
        return dataclasses.replace(
            self, model=m,
            n_ctx=self.n_ctx if n_ctx is None else n_ctx,
            n_prompt=self.n_prompt if n_prompt is None else n_prompt,
            key=f"{self.key}-L{m.n_layers}-N{n_ctx or self.n_ctx}-P{self.n_prompt if n_prompt is None else n_prompt}")


TINY = ModelConfig("tiny", 2, 256, 4, 2, 64, 688, 1024, 1e4, 16)
M1B = ModelConfig("llama-1b", 16, 2048, 32, 8, 64, 8192, 128256, 5e5, 256)
M3B = ModelConfig("llama-3b", 28, 3072, 24, 8, 128, 8192, 128256, 5e5, 256)
M1P5B = ModelConfig("qwen-1.5b", 28, 1536, 12, 2, 128, 8960, 151936, 5e5, 256)
M8B = ModelConfig("llama-8b", 32, 4096, 32, 8, 128, 14336, 128256, 5e5, 256)

WORKLOADS = {
    "tiny": Workload("tiny", 1, TINY, 128, 0, "random-half-drop",
                     "tiny 2L d256, 128-token context, 50% of KV chunks dropped at random"),
    "1b": Workload("1b", 2, M1B, 2048, 0, "all-drop",
                   "1B-class 16L d2048, 2048-token context fully dropped (weights resident)"),
    "3b": Workload("3b", 3, M3B, 8192, 64, "back-half-layers-drop",
                   "3B-class 28L d3072, 8192-token context, KV of last 14 layers dropped, 64-token prompt"),
    "1p5b": Workload("1p5b", 4, M1P5B, 16384, 0, "hybrid-40swap-30drop",
                     "1.5B-class 28L d1536, 16384-token context, 40% KV swapped / 30% dropped / 30% resident"),
    "8b": Workload("8b", 5, M8B, 32768, 128, "backward-out-75pct-weights-swap",
                   "8B-class 32L d4096, 32768-token context, last 8 weight layers + 50% KV swapped, "
                   "25% KV dropped, 128-token prompt"),
}
ORDERED_KEYS = ["tiny", "1b", "3b", "1p5b", "8b"]


# ----------------------------------------------------------------------------- blob layout

def tensor_shapes(m: ModelConfig) -> List[Tuple[str, int, int, int]]:
    """(name, layer, out, in) for every tensor in blob order."""
    out = []
    for l in range(m.n_layers):
        out += [("wq", l, m.dq, m.d_model), ("wk", l, m.dkv, m.d_model), ("wv", l, m.dkv, m.d_model),
                ("wo", l, m.d_model, m.dq), ("wg", l, m.d_ffn, m.d_model), ("wu", l, m.d_ffn, m.d_model),
                ("wd", l, m.d_model, m.d_ffn)]
    out += [("emb", -1, m.vocab, m.d_model), ("lm", -1, m.vocab, m.d_model)]
    return out


def q4_0_nbytes(rows: int, cols: int) -> int:
    return rows * ((cols + 31) // 32) * 18


def blob_nbytes(m: ModelConfig) -> int:
    return sum(q4_0_nbytes(r, c) for _, _, r, c in tensor_shapes(m))


# ----------------------------------------------------------------------------- C generator

_lib = None


def _synth_lib():
    global _lib
    if _lib is not None:
        return _lib
    if (not os.path.exists(_SYNTH_LIB)
            or os.path.getmtime(_SYNTH_LIB) < os.path.getmtime(_SYNTH_SRC)):
        build_synth()
    lib = ctypes.CDLL(_SYNTH_LIB)
    u32, i64, u64 = ctypes.c_uint32, ctypes.c_int64, ctypes.c_uint64
    vp = ctypes.c_void_p
    lib.mz_synth_q4_0.argtypes = [u32, u32, i64, i64, ctypes.c_float, vp]
    lib.mz_synth_normal.argtypes = [u32, u32, u64, u64, ctypes.c_float, vp]
    lib.mz_encode_q4_0.argtypes = [vp, i64, i64, vp]
    lib.mz_f32_to_f16.argtypes = [vp, vp, u64]
    lib.mz_philox4x32_10.argtypes = [vp, vp, vp]
    _lib = lib
    return lib


def build_synth() -> str:
    """Compile the input generator (plain C, OpenMP)."""
    tmp = _SYNTH_LIB + ".tmp"
    subprocess.check_call(["gcc", "-O3", "-fopenmp", "-shared", "-fPIC", "-Wall", "-o", tmp,
                           _SYNTH_SRC, "-lm"])
    os.replace(tmp, _SYNTH_LIB)
    return _SYNTH_LIB


def philox4x32_10(ctr, key) -> np.ndarray:
    c = np.ascontiguousarray(ctr, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.empty(4, np.uint32)
    _synth_lib().mz_philox4x32_10(c.ctypes.data, k.ctypes.data, out.ctypes.data)
    return out


def normals(seed: int, tensor_id: int, start: int, n: int, std: float = 1.0) -> np.ndarray:
    out = np.empty(n, np.float32)
    _synth_lib().mz_synth_normal(seed, tensor_id, start, n, std, out.ctypes.data)
    return out


def encode_q4_0(x: np.ndarray) -> np.ndarray:
    """Encode float32 [rows, cols] as Q4_0 bytes [rows, ceil(cols/32)*18]."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    rows, cols = x.shape
    out = np.empty((rows, ((cols + 31) // 32) * 18), np.uint8)
    _synth_lib().mz_encode_q4_0(x.ctypes.data, rows, cols, out.ctypes.data)
    return out


def synth_q4_0(seed: int, tensor_id: int, rows: int, cols: int, std: float = 0.02,
               out: Optional[np.ndarray] = None) -> np.ndarray:
    n = q4_0_nbytes(rows, cols)
    if out is None:
        out = np.empty(n, np.uint8)
    assert out.nbytes == n and out.flags["C_CONTIGUOUS"]
    _synth_lib().mz_synth_q4_0(seed, tensor_id, rows, cols, std, out.ctypes.data)
    return out


def make_blob(w: Workload, std: float = 0.02) -> np.ndarray:
    """The full Q4_0 model blob for a workload (seeded by its config id)."""
    m = w.model
    blob = np.empty(blob_nbytes(m), np.uint8)
    off = 0
    for tid, (_, _, rows, cols) in enumerate(tensor_shapes(m)):
        n = q4_0_nbytes(rows, cols)
        synth_q4_0(w.config_id, tid, rows, cols, std, out=blob[off:off + n])
        off += n
    return blob


# ----------------------------------------------------------------------------- tokens & plans

def make_tokens(w: Workload) -> Tuple[np.ndarray, np.ndarray]:
    """Uniform random context ids (seed 0) and prompt ids (seed 1)."""
    ctx = np.random.default_rng(0).integers(0, w.model.vocab, w.n_ctx, dtype=np.int64).astype(np.int32)
    prm = np.random.default_rng(1).integers(0, w.model.vocab, w.n_prompt, dtype=np.int64).astype(np.int32)
    return ctx, prm


@dataclasses.dataclass
class Plan:
    kv_state: np.ndarray            # uint8 [L, n_chunks]
    w_state: np.ndarray             # uint8 [L]
    order: Optional[np.ndarray] = None   # int32 unit ids, None = backward-out

    def counts(self):
        return {s: int((self.kv_state == v).sum()) for s, v in (("res", RES), ("swap", SWAP), ("drop", DROP))}


def backward_out_units(n_layers: int, n_chunks: int) -> List[Tuple[int, int]]:
    """KV units in backward-out order: last layer first, last chunk first (Sec. 4.4)."""
    return [(l, c) for l in range(n_layers - 1, -1, -1) for c in range(n_chunks - 1, -1, -1)]


def make_plan(w: Workload) -> Plan:
    L, nc = w.model.n_layers, w.n_chunks
    kv = np.zeros((L, nc), np.uint8)
    ws = np.zeros(L, np.uint8)
    total = L * nc
    rule = w.plan_rule
    if rule == "random-half-drop":
        idx = np.random.default_rng(0).permutation(total)[: total // 2]
        kv.reshape(-1)[idx] = DROP
    elif rule == "all-drop":
        kv[:] = DROP
    elif rule == "back-half-layers-drop":
        kv[L // 2:] = DROP
    elif rule == "hybrid-40swap-30drop":
        n_swap, n_drop = int(round(0.4 * total)), int(round(0.3 * total))
        perm = np.random.default_rng(0).permutation(total)
        kv.reshape(-1)[perm[:n_swap]] = SWAP
        kv.reshape(-1)[perm[n_swap:n_swap + n_drop]] = DROP
    elif rule == "backward-out-75pct-weights-swap":
        n_ev = int(round(0.75 * total))
        for r, (l, c) in enumerate(backward_out_units(L, nc)[:n_ev]):
            kv[l, c] = DROP if r % 3 == 2 else SWAP
        ws[L - L // 4:] = SWAP
    else:
        raise ValueError(f"unknown plan rule {rule}")
    return Plan(kv, ws)


def random_plan(n_layers: int, n_chunks: int, p_swap: float, p_drop: float, seed: int,
                w_swap: float = 0.0, w_drop: float = 0.0) -> Plan:
    """Independent per-unit states, for tests."""
    rng = np.random.default_rng(seed)
    u = rng.random((n_layers, n_chunks))
    kv = np.where(u < p_swap, SWAP, np.where(u < p_swap + p_drop, DROP, RES)).astype(np.uint8)
    v = rng.random(n_layers)
    ws = np.where(v < w_swap, SWAP, np.where(v < w_swap + w_drop, DROP, RES)).astype(np.uint8)
    return Plan(kv, ws)
