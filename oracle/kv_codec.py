"""8-bit group-wise KV codec for the swap path (TEST INFRASTRUCTURE ONLY, like
the rest of oracle/; shares no code with the library's codec).

The paper compresses swapped KV chunks with 8-bit quantization as its default
codec (Sec. 5, after FlexGen's group-wise scheme) and notes that repeated
compression and decompression does not accumulate error (Sec. 6).  Definition
used here, on a flat sequence of IEEE half values whose length is a multiple
of 64, taken in groups of 64 consecutive values (for a KV chunk: its K
token-major, then its V dimension-major, the order of the device slot):

    mn, mx = min, max of the group (exact in fp32)
    d      = half( fp32(mx - mn) / 255 )           step, rounded to nearest even
    m      = mn                                     (a half value already)
    q_i    = 0 if d == 0 else clamp(rint(fp32(x_i - m) / fp32(d)), 0, 255)
    x^_i   = half( fp32(q_i) * fp32(d) + fp32(m) )  (the product is exact)

Every division is one correctly rounded fp32 division and rint rounds half to
even, so an implementation following these steps reaches the same codes bit
for bit.  Stored layout for n values: n code bytes, then per group the halves
(m, d): n + n / 16 bytes.
"""

from __future__ import annotations

import numpy as np

GROUP = 64


def compressed_bytes(n: int) -> int:
    return n + (n // GROUP) * 4


def compress(x: np.ndarray) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float16).reshape(-1)
    if x.size % GROUP:
        raise ValueError("length must be a multiple of 64")
    g = x.reshape(-1, GROUP).astype(np.float32)
    mn = g.min(axis=1)
    mx = g.max(axis=1)
    d = ((mx - mn) / np.float32(255.0)).astype(np.float16)
    d32 = d.astype(np.float32)
    safe = np.where(d32 == 0, np.float32(1.0), d32)
    q = np.rint((g - mn[:, None]) / safe[:, None])
    q = np.where(d32[:, None] == 0, np.float32(0.0), q)
    q = np.clip(q, 0, 255).astype(np.uint8)
    params = np.stack([mn.astype(np.float16), d], axis=1)          # (m, d) per group
    return np.concatenate([q.reshape(-1), params.reshape(-1).view(np.uint8)])


def decompress(blob: np.ndarray, n: int) -> np.ndarray:
    blob = np.ascontiguousarray(blob, dtype=np.uint8).reshape(-1)
    if blob.size != compressed_bytes(n):
        raise ValueError("compressed size does not match n")
    q = blob[:n].reshape(-1, GROUP).astype(np.float32)
    params = blob[n:].view(np.float16).reshape(-1, 2).astype(np.float32)
    m, d = params[:, 0:1], params[:, 1:2]
    return (q * d + m).astype(np.float32).astype(np.float16).reshape(-1)


def chunk_device_order(k: np.ndarray, v: np.ndarray) -> np.ndarray:
    """K [C][dkv] and V [C][dkv] (exchange layout) -> the device slot's value
    order: K token-major, then V dimension-major."""
    return np.concatenate([np.ascontiguousarray(k, np.float16).reshape(-1),
                           np.ascontiguousarray(np.asarray(v, np.float16).T).reshape(-1)])


def chunk_from_device_order(flat: np.ndarray, C: int, dkv: int):
    k = flat[:C * dkv].reshape(C, dkv)
    v = flat[C * dkv:].reshape(dkv, C).T.copy()
    return k, v


def roundtrip_chunk(k: np.ndarray, v: np.ndarray):
    """What a chunk looks like after one swap through the codec."""
    C, dkv = np.asarray(k).shape
    flat = chunk_device_order(k, v)
    return chunk_from_device_order(decompress(compress(flat), flat.size), C, dkv)
