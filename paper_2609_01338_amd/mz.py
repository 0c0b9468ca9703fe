"""Python binding of libmz (ctypes).  Argument marshalling only: every step of
the restore-and-prefill path runs in the library's HIP kernels.  Function names
match the C ABI in include/mz.h; a non-zero status raises MzError.

The library is loaded from this package directory; a missing library is an
error (there is no fallback path).
"""

from __future__ import annotations

import ctypes
import json
import os
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmz.so")

MZ_OK, MZ_EINVAL, MZ_ENOMEM, MZ_EHIP, MZ_ESTATE = 0, -1, -2, -3, -4
MZ_RES, MZ_SWAP, MZ_DROP = 0, 1, 2
STATUS_NAMES = {0: "MZ_OK", -1: "MZ_EINVAL", -2: "MZ_ENOMEM", -3: "MZ_EHIP", -4: "MZ_ESTATE"}


class MzError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


class mz_model_cfg(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32),
                ("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("d_ffn", ctypes.c_int32), ("vocab", ctypes.c_int32),
                ("chunk_tokens", ctypes.c_int32), ("max_ctx", ctypes.c_int32),
                ("rope_theta", ctypes.c_float), ("rms_eps", ctypes.c_float)]


class mz_evict_plan(ctypes.Structure):
    _fields_ = [("kv_state", ctypes.c_void_p), ("n_layers", ctypes.c_int32),
                ("n_chunks", ctypes.c_int32), ("w_state", ctypes.c_void_p),
                ("order", ctypes.c_void_p), ("n_order", ctypes.c_int32)]


class mz_evict_request(ctypes.Structure):
    _fields_ = [("n_ctx", ctypes.c_int32), ("n_prompt", ctypes.c_int32), ("n_kv_evict", ctypes.c_int32),
                ("n_w_evict", ctypes.c_int32), ("order", ctypes.c_int32), ("placement", ctypes.c_int32),
                ("seed", ctypes.c_uint64), ("link_bytes_per_s", ctypes.c_double),
                ("recompute_flops_per_s", ctypes.c_double), ("kv_codec", ctypes.c_int32)]


class mz_evict_size_request(ctypes.Structure):
    _fields_ = [("bytes", ctypes.c_int64), ("n_prompt", ctypes.c_int32), ("n_w_total", ctypes.c_int32),
                ("link_bytes_per_s", ctypes.c_double), ("recompute_flops_per_s", ctypes.c_double),
                ("kv_codec", ctypes.c_int32), ("rule", ctypes.c_int32)]


class mz_q4_gemm_args(ctypes.Structure):
    _fields_ = [("a_rows", ctypes.c_void_p), ("work_queues", ctypes.c_void_p), ("workspace", ctypes.c_void_p),
                ("workspace_bytes", ctypes.c_int64), ("pos", ctypes.c_void_p), ("rope_cs", ctypes.c_void_p),
                ("kv_off", ctypes.c_void_p), ("slab", ctypes.c_void_p), ("head_dim", ctypes.c_int32),
                ("n_valid", ctypes.c_int32), ("chunk_tokens", ctypes.c_int32)]


SIZE_RULES = {"paper": 0, "total": 1}
STAGES = ("kv-only", "kv-and-w", "w-only", "exhausted")
_INFO_KEYS = ("released", "T", "stage", "link_s", "recompute_s", "n_kv", "n_w", "reached")


def _size_info(info: np.ndarray) -> dict:
    d = dict(zip(_INFO_KEYS, (float(v) for v in info)))
    for k in ("released", "T", "n_kv", "n_w"):
        d[k] = int(d[k])
    d["stage"] = STAGES[int(d["stage"])]
    d["reached"] = bool(d["reached"])
    return d


ORDERS = {"backward-out": 0, "forward-out": 1, "random-out": 2, "token-aligned": 3}
PLACEMENTS = {"balanced": 0, "all-swap": 1, "all-drop": 2, "interleave-2-1": 3}

_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run paper_2609_01338_amd.build")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    sigs = {
        "mz_load_model": ([ctypes.POINTER(mz_model_cfg), vp, sz, i32, ctypes.POINTER(vp)], i32),
        "mz_prefill_context": ([vp, vp, i32], i32),
        "mz_set_context": ([vp, vp, i32], i32),
        "mz_truncate_context": ([vp, i32], i32),
        "mz_import_kv": ([vp, i32, i32, vp, vp], i32),
        "mz_read_kv": ([vp, i32, i32, vp, vp], i32),
        "mz_evict": ([vp, ctypes.POINTER(mz_evict_plan)], i32),
        "mz_restore_and_prefill": ([vp, vp, i32], i32),
        "mz_first_token": ([vp, vp, vp], i32),
        "mz_set_option": ([vp, ctypes.c_char_p, i64], i32),
        "mz_generate": ([vp, i32, i32, vp], i32),
        "mz_stats": ([vp, ctypes.c_char_p, sz], i32),
        "mz_last_error": ([vp], ctypes.c_char_p),
        "mz_free": ([vp], None),
        "mz_version": ([], ctypes.c_char_p),
        "mz_plan_rows": ([ctypes.POINTER(mz_model_cfg), vp, i32, i32, i32, vp, vp, vp, i64], i32),
        "mz_q4_gemm_packed_bytes": ([i32, i32], i64),
        "mz_q4_gemm_pack": ([vp, vp, i32, i32, vp], i32),
        "mz_q4_gemm": ([vp, i32, i32, i32, vp, i32, vp, vp], i32),
        "mz_attention": ([vp, vp, i32, vp, vp, i32, i32, i32, i32, i32, vp, vp], i32),
        "mz_attention_queued": ([vp, vp, i32, vp, vp, i32, i32, i32, i32, i32, vp, vp, vp], i32),
        "mz_q4_gemm_queued": ([vp, i32, i32, i32, vp, i32, vp, vp, vp], i32),
        "mz_q4_gemm_ex": ([vp, i32, i32, i32, vp, i32, ctypes.POINTER(mz_q4_gemm_args), vp, vp], i32),
        "mz_q4_gemv": ([vp, i32, vp, i32, i32, ctypes.POINTER(mz_q4_gemm_args), vp, ctypes.c_float, vp, vp], i32),
        "mz_rmsnorm": ([vp, i32, i32, ctypes.c_float, vp, vp], i32),
        "mz_probe_ceilings": ([i32, ctypes.c_char_p, sz], i32),
        "mz_plan_evict": ([ctypes.POINTER(mz_model_cfg), ctypes.POINTER(mz_evict_request), vp, vp, vp], i32),
        "mz_kv_compress": ([vp, i64, vp, vp], i32),
        "mz_kv_decompress": ([vp, i64, vp, vp], i32),
        "mz_q4_gemm_split": ([vp, i32, i32, i32, vp, i32, vp, i32, vp, i64, vp], i32),
        "mz_q4_gemm_split_workspace_bytes": ([i32, i32, i32], i64),
        "mz_q4_gemm_split_noalloc": ([vp, i32, i32, i32, vp, i32, vp, i32, vp], i32),
        "mz_q4_gemm_auto_splits": ([i32, i32, i32, i64], i32),
        "mz_q4_gemm_long_k_splits": ([i32, i32, i32, i64], i32),
        "mz_attention_split": ([vp, vp, i32, i32, vp, vp, i32, i32, i32, i32, i32, i32, vp, i64, vp, vp], i32),
        "mz_attention_split_workspace_bytes": ([i32, i32, i32, i32], i64),
        "mz_attention_auto_splits": ([i32, i32, i32, i32, i32, i64], i32),
        "mz_plan_evict_size": ([ctypes.POINTER(mz_model_cfg), i32, ctypes.POINTER(mz_evict_size_request),
                                vp, vp, vp, vp, vp, vp], i32),
        "mz_evict_size": ([vp, ctypes.POINTER(mz_evict_size_request), vp], i32),
    }
    for name, (args, res) in sigs.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = res
    _lib = L
    return L


def _check(status: int, ctx=None):
    if status != MZ_OK:
        msg = lib().mz_last_error(ctx)
        raise MzError(status, msg.decode() if msg else "")


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data


def make_cfg(model, max_ctx: int) -> mz_model_cfg:
    """mz_model_cfg from any object with the model-shape attributes."""
    return mz_model_cfg(model.n_layers, model.d_model, model.n_q_heads, model.n_kv_heads,
                        model.head_dim, model.d_ffn, model.vocab, model.chunk_tokens, max_ctx,
                        float(model.rope_theta), float(model.rms_eps))


# ----------------------------------------------------------------------------- model level

def mz_version() -> str:
    return lib().mz_version().decode()


def mz_load_model(cfg: mz_model_cfg, blob: np.ndarray, device: int = 0) -> ctypes.c_void_p:
    blob = np.ascontiguousarray(blob, dtype=np.uint8)
    out = ctypes.c_void_p()
    _check(lib().mz_load_model(ctypes.byref(cfg), blob.ctypes.data, blob.nbytes, device,
                               ctypes.byref(out)), None)
    return out


def mz_free(ctx) -> None:
    lib().mz_free(ctx)


def mz_prefill_context(ctx, tokens: np.ndarray) -> None:
    t = np.ascontiguousarray(tokens, dtype=np.int32)
    _check(lib().mz_prefill_context(ctx, _ptr(t), t.size), ctx)


def mz_set_context(ctx, tokens: np.ndarray) -> None:
    t = np.ascontiguousarray(tokens, dtype=np.int32)
    _check(lib().mz_set_context(ctx, _ptr(t), t.size), ctx)


def mz_truncate_context(ctx, n: int) -> None:
    _check(lib().mz_truncate_context(ctx, n), ctx)


def mz_import_kv(ctx, layer: int, chunk: int, k: np.ndarray, v: np.ndarray) -> None:
    k = np.ascontiguousarray(k, dtype=np.float16)
    v = np.ascontiguousarray(v, dtype=np.float16)
    _check(lib().mz_import_kv(ctx, layer, chunk, k.ctypes.data, v.ctypes.data), ctx)


def mz_read_kv(ctx, layer: int, chunk: int, chunk_tokens: int, dkv: int):
    k = np.empty((chunk_tokens, dkv), np.float16)
    v = np.empty((chunk_tokens, dkv), np.float16)
    _check(lib().mz_read_kv(ctx, layer, chunk, k.ctypes.data, v.ctypes.data), ctx)
    return k, v


def mz_evict(ctx, kv_state: np.ndarray, w_state: Optional[np.ndarray] = None,
             order: Optional[np.ndarray] = None) -> None:
    kv = np.ascontiguousarray(kv_state, dtype=np.uint8)
    ws = None if w_state is None else np.ascontiguousarray(w_state, dtype=np.uint8)
    od = None if order is None else np.ascontiguousarray(order, dtype=np.int32)
    plan = mz_evict_plan(kv.ctypes.data, kv.shape[0], kv.shape[1], _ptr(ws), _ptr(od),
                         0 if od is None else od.size)
    _check(lib().mz_evict(ctx, ctypes.byref(plan)), ctx)


def mz_evict_size(ctx, nbytes: int, link_bytes_per_s: float, recompute_flops_per_s: float,
                  n_w_total: int, n_prompt: int = 0, rule: str = "paper") -> dict:
    """Release at least nbytes of device memory by the hybrid-swap policy;
    returns {released, T, stage, link_s, recompute_s, n_kv, n_w, reached}."""
    req = mz_evict_size_request(int(nbytes), int(n_prompt), int(n_w_total), float(link_bytes_per_s),
                                float(recompute_flops_per_s), 0, SIZE_RULES[rule])
    info = np.zeros(8, np.float64)
    _check(lib().mz_evict_size(ctx, ctypes.byref(req), info.ctypes.data), ctx)
    return _size_info(info)


def mz_restore_and_prefill(ctx, prompt: Optional[np.ndarray] = None) -> None:
    p = np.zeros(0, np.int32) if prompt is None else np.ascontiguousarray(prompt, dtype=np.int32)
    _check(lib().mz_restore_and_prefill(ctx, _ptr(p) if p.size else None, p.size), ctx)


def mz_first_token(ctx, vocab: Optional[int] = None):
    """Returns the token, and the logits when vocab is given."""
    tok = ctypes.c_int32()
    logits = None if vocab is None else np.empty(vocab, np.float32)
    _check(lib().mz_first_token(ctx, ctypes.byref(tok), _ptr(logits)), ctx)
    return (tok.value, logits) if vocab is not None else tok.value


def mz_generate(ctx, token: int, n: int) -> np.ndarray:
    """Append token and decode n more tokens greedily."""
    out = np.zeros(max(n, 1), np.int32)
    _check(lib().mz_generate(ctx, int(token), int(n), out.ctypes.data), ctx)
    return out[:n]


def mz_set_option(ctx, key: str, value: int) -> None:
    _check(lib().mz_set_option(ctx, key.encode(), int(value)), ctx)


def mz_stats(ctx) -> dict:
    buf = ctypes.create_string_buffer(1 << 16)
    _check(lib().mz_stats(ctx, buf, len(buf)), ctx)
    return json.loads(buf.value.decode())


def mz_last_error(ctx=None) -> str:
    m = lib().mz_last_error(ctx)
    return m.decode() if m else ""


# ----------------------------------------------------------------------------- host helpers

def mz_plan_evict(cfg: mz_model_cfg, n_ctx: int, n_prompt: int, n_kv_evict: int, n_w_evict: int,
                  order: str = "backward-out", placement: str = "balanced", seed: int = 0,
                  link_bytes_per_s: float = 0.0, recompute_flops_per_s: float = 0.0, kv_codec: bool = False):
    """Eviction plan (kv_state [L][n_chunks] uint8, w_state [L] uint8) and the
    estimate dict {swap_bytes, restore_flops, link_s, recompute_s, pipeline_s}."""
    L = cfg.n_layers
    nc = (n_ctx + cfg.chunk_tokens - 1) // cfg.chunk_tokens
    req = mz_evict_request(n_ctx, n_prompt, n_kv_evict, n_w_evict, ORDERS[order], PLACEMENTS[placement],
                           seed, link_bytes_per_s, recompute_flops_per_s, int(kv_codec))
    kv = np.empty((L, nc), np.uint8)
    ws = np.empty(L, np.uint8)
    est = np.empty(5, np.float64)
    _check(lib().mz_plan_evict(ctypes.byref(cfg), ctypes.byref(req), kv.ctypes.data, ws.ctypes.data,
                               est.ctypes.data), None)
    return kv, ws, {"swap_bytes": est[0], "restore_flops": est[1], "link_s": est[2], "recompute_s": est[3],
                    "pipeline_s": est[4]}


def mz_plan_evict_size(cfg: mz_model_cfg, n_ctx: int, kv_state: np.ndarray, w_state: np.ndarray, nbytes: int,
                       link_bytes_per_s: float, recompute_flops_per_s: float, n_w_total: int,
                       n_prompt: int = 0, kv_codec: bool = False, rule: str = "paper"):
    """Next increment of size-driven eviction from the given states:
    (kv_state, w_state updated copies, evicted unit ids in order, their
    stages, info dict)."""
    kv = np.array(kv_state, dtype=np.uint8, order="C", copy=True)
    ws = np.array(w_state, dtype=np.uint8, order="C", copy=True)
    L, nc = kv.shape
    order = np.empty(L * (nc + 1), np.int32)
    stage = np.empty(L * (nc + 1), np.int32)
    n = ctypes.c_int32()
    info = np.zeros(8, np.float64)
    req = mz_evict_size_request(int(nbytes), int(n_prompt), int(n_w_total), float(link_bytes_per_s),
                                float(recompute_flops_per_s), int(kv_codec), SIZE_RULES[rule])
    _check(lib().mz_plan_evict_size(ctypes.byref(cfg), n_ctx, ctypes.byref(req), kv.ctypes.data, ws.ctypes.data,
                                    order.ctypes.data, stage.ctypes.data, ctypes.byref(n), info.ctypes.data),
           None)
    return kv, ws, order[:n.value].copy(), stage[:n.value].copy(), _size_info(info)


def mz_plan_rows(cfg: mz_model_cfg, kv_state: np.ndarray, n_ctx: int, n_prompt: int,
                 with_rows: bool = True):
    kv = np.ascontiguousarray(kv_state, dtype=np.uint8)
    L = cfg.n_layers
    nR = np.empty(L, np.int32)
    nD = np.empty(L, np.int32)
    cap = L * (n_ctx + n_prompt) if with_rows else 0
    rows = np.empty(max(cap, 1), np.int32) if with_rows else None
    _check(lib().mz_plan_rows(ctypes.byref(cfg), kv.ctypes.data, kv.shape[1], n_ctx, n_prompt,
                              nR.ctypes.data, nD.ctypes.data, _ptr(rows), cap), None)
    if not with_rows:
        return nR, nD, None
    R, o = [], 0
    for l in range(L):
        R.append(rows[o:o + nR[l]].copy())
        o += nR[l]
    return nR, nD, R


def mz_q4_gemm_packed_bytes(n: int, k: int) -> int:
    return int(lib().mz_q4_gemm_packed_bytes(n, k))


def mz_q4_gemm_pack(w: np.ndarray, n: int, k: int, w_up: Optional[np.ndarray] = None) -> np.ndarray:
    w = np.ascontiguousarray(w, dtype=np.uint8)
    if w_up is None:
        out = np.empty(mz_q4_gemm_packed_bytes(n, k), np.uint8)
    else:
        w_up = np.ascontiguousarray(w_up, dtype=np.uint8)
        n128 = (n + 127) // 128 * 128
        out = np.empty(mz_q4_gemm_packed_bytes(2 * n128, k), np.uint8)
    _check(lib().mz_q4_gemm_pack(w.ctypes.data, _ptr(w_up), n, k, out.ctypes.data), None)
    return out


# ----------------------------------------------------------------------------- kernel level
# Device pointers are integers (e.g. torch.Tensor.data_ptr()); stream is a
# hipStream_t as an integer or None.

def mz_q4_gemm(x_ptr: int, m: int, n_pad: int, k: int, w_ptr: int, epilogue: int, y_ptr: int,
               stream: Optional[int] = None) -> None:
    _check(lib().mz_q4_gemm(x_ptr, m, n_pad, k, w_ptr, epilogue, y_ptr, stream), None)


def mz_q4_gemm_queued(x_ptr: int, m: int, n_pad: int, k: int, w_ptr: int, epilogue: int, y_ptr: int,
                      queues_ptr: int, stream: Optional[int] = None) -> None:
    _check(lib().mz_q4_gemm_queued(x_ptr, m, n_pad, k, w_ptr, epilogue, y_ptr, queues_ptr, stream), None)


def mz_q4_gemm_ex(x_ptr: int, m: int, n_pad: int, k: int, w_ptr: int, epilogue: int, y_ptr: Optional[int],
                  stream: Optional[int] = None, a_rows: int = 0, work_queues: int = 0, workspace: int = 0,
                  workspace_bytes: int = 0, pos: int = 0, rope_cs: int = 0, kv_off: int = 0, slab: int = 0,
                  head_dim: int = 0, n_valid: int = 0, chunk_tokens: int = 0) -> None:
    """Device pointers as integers (0: absent)."""
    a = mz_q4_gemm_args(a_rows or None, work_queues or None, workspace or None, workspace_bytes, pos or None,
                        rope_cs or None, kv_off or None, slab or None, head_dim, n_valid, chunk_tokens)
    _check(lib().mz_q4_gemm_ex(x_ptr, m, n_pad, k, w_ptr, epilogue, ctypes.byref(a), y_ptr or None, stream), None)


def mz_q4_gemv(x_ptr: Optional[int], k: int, w_ptr: int, n_pad: int, epilogue: int, y_ptr: Optional[int],
               stream: Optional[int] = None, a_rows: int = 0, h_norm: int = 0, eps: float = 0.0, pos: int = 0,
               rope_cs: int = 0, kv_off: int = 0, slab: int = 0, head_dim: int = 0, n_valid: int = 0,
               chunk_tokens: int = 0) -> None:
    """Device pointers as integers (0: absent)."""
    a = mz_q4_gemm_args(a_rows or None, None, None, 0, pos or None, rope_cs or None, kv_off or None, slab or None,
                        head_dim, n_valid, chunk_tokens)
    _check(lib().mz_q4_gemv(x_ptr or None, k, w_ptr, n_pad, epilogue, ctypes.byref(a), h_norm or None, eps,
                            y_ptr or None, stream), None)


def mz_attention(q_ptr: int, qpos_ptr: int, m: int, slab_ptr: int, table_ptr: int, n_table: int,
                 chunk_tokens: int, n_q: int, n_kv: int, head_dim: int, out_ptr: int,
                 stream: Optional[int] = None) -> None:
    _check(lib().mz_attention(q_ptr, qpos_ptr, m, slab_ptr, table_ptr, n_table, chunk_tokens, n_q,
                              n_kv, head_dim, out_ptr, stream), None)


def mz_attention_queued(q_ptr: int, qpos_ptr: int, m: int, slab_ptr: int, table_ptr: int, n_table: int,
                        chunk_tokens: int, n_q: int, n_kv: int, head_dim: int, out_ptr: int, queues_ptr: int,
                        stream: Optional[int] = None) -> None:
    _check(lib().mz_attention_queued(q_ptr, qpos_ptr, m, slab_ptr, table_ptr, n_table, chunk_tokens, n_q,
                                     n_kv, head_dim, out_ptr, queues_ptr, stream), None)


def mz_q4_gemm_split(x_ptr: int, m: int, n_pad: int, k: int, w_ptr: int, epilogue: int, y_ptr: int,
                     n_split: int, ws_ptr: int, ws_bytes: int, stream: Optional[int] = None) -> None:
    _check(lib().mz_q4_gemm_split(x_ptr, m, n_pad, k, w_ptr, epilogue, y_ptr, n_split, ws_ptr, ws_bytes, stream),
           None)


NOALLOC_SCRATCH_BYTES = 32 * 1024 * 1024


def mz_q4_gemm_split_noalloc(x_ptr: int, m: int, n_pad: int, k: int, w_ptr: int, epilogue: int, y_ptr: int,
                             n_split: int, stream: Optional[int] = None) -> None:
    _check(lib().mz_q4_gemm_split_noalloc(x_ptr, m, n_pad, k, w_ptr, epilogue, y_ptr, n_split, stream), None)


def mz_q4_gemm_split_workspace_bytes(m: int, n_pad: int, n_split: int) -> int:
    return int(lib().mz_q4_gemm_split_workspace_bytes(m, n_pad, n_split))


def mz_q4_gemm_auto_splits(m: int, n_pad: int, k: int, ws_bytes: int) -> int:
    return int(lib().mz_q4_gemm_auto_splits(m, n_pad, k, ws_bytes))


def mz_q4_gemm_long_k_splits(m: int, n_pad: int, k: int, ws_bytes: int) -> int:
    return int(lib().mz_q4_gemm_long_k_splits(m, n_pad, k, ws_bytes))


def mz_attention_split(q_ptr: int, qpos_ptr: int, m: int, max_pos: int, slab_ptr: int, table_ptr: int,
                       n_table: int, chunk_tokens: int, n_q: int, n_kv: int, head_dim: int, n_split: int,
                       ws_ptr: int, ws_bytes: int, out_ptr: int, stream: Optional[int] = None) -> None:
    _check(lib().mz_attention_split(q_ptr, qpos_ptr, m, max_pos, slab_ptr, table_ptr, n_table, chunk_tokens, n_q,
                                    n_kv, head_dim, n_split, ws_ptr, ws_bytes, out_ptr, stream), None)


def mz_attention_split_workspace_bytes(m: int, n_q: int, head_dim: int, n_split: int) -> int:
    return int(lib().mz_attention_split_workspace_bytes(m, n_q, head_dim, n_split))


def mz_attention_auto_splits(m: int, max_pos: int, n_q: int, n_kv: int, head_dim: int, ws_bytes: int) -> int:
    return int(lib().mz_attention_auto_splits(m, max_pos, n_q, n_kv, head_dim, ws_bytes))


def mz_rmsnorm(h_ptr: int, m: int, d: int, eps: float, x_ptr: int, stream: Optional[int] = None) -> None:
    _check(lib().mz_rmsnorm(h_ptr, m, d, eps, x_ptr, stream), None)


def mz_kv_compress(src_ptr: int, n_halves: int, out_ptr: int, stream: Optional[int] = None) -> None:
    _check(lib().mz_kv_compress(src_ptr, n_halves, out_ptr, stream), None)


def mz_kv_decompress(in_ptr: int, n_halves: int, dst_ptr: int, stream: Optional[int] = None) -> None:
    _check(lib().mz_kv_decompress(in_ptr, n_halves, dst_ptr, stream), None)


def mz_probe_ceilings(device: int = 0) -> dict:
    buf = ctypes.create_string_buffer(1024)
    _check(lib().mz_probe_ceilings(device, buf, len(buf)), None)
    return json.loads(buf.value.decode())


class Engine:
    """Convenience owner of one context (closes it on exit)."""

    def __init__(self, model, blob: np.ndarray, max_ctx: int, device: int = 0):
        self.model = model
        self.cfg = make_cfg(model, max_ctx)
        self.ctx = mz_load_model(self.cfg, blob, device)

    def close(self):
        if self.ctx:
            mz_free(self.ctx)
            self.ctx = None

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
