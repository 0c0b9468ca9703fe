// Memory-bound kernels of the restore-and-prefill path (gfx950): RMSNorm,
// rotary embedding with KV scatter into chunk slots, embedding gather with
// Q4_0 dequantization, row compaction, and the output head with argmax.
#include "mz_kernels.h"
#include "rope.h"
#include "rownorm.h"

namespace mzk {
namespace {

// One 256-thread block per row; d % 4 == 0.  The row is read once: each
// thread keeps its up to kRowNormRegs float4 pieces in registers between the
// sum of squares and the scaled store (rows longer than 256 * kRowNormRegs * 4
// read the rest twice).
__global__ __launch_bounds__(256) void rmsnorm_kernel(const float* __restrict__ h, int d, float eps,
                                                      _Float16* __restrict__ x) {
  __shared__ float red[4];
  const int row = blockIdx.x;
  const int n4 = d / 4;
  const float* hrow = h + (size_t)row * d;
  float4 v[kRowNormRegs];
  const float r = row_inv_rms(hrow, d, eps, v, red);
  typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
  f16x4* xr = reinterpret_cast<f16x4*>(x + (size_t)row * d);
#pragma unroll
  for (int k = 0; k < kRowNormRegs; ++k) {
    const int i = threadIdx.x + k * 256;
    if (i < n4)
      xr[i] = f16x4{norm_to_f16(v[k].x, r), norm_to_f16(v[k].y, r), norm_to_f16(v[k].z, r), norm_to_f16(v[k].w, r)};
  }
  const float4* hr = reinterpret_cast<const float4*>(hrow);
  for (int i = threadIdx.x + kRowNormRegs * 256; i < n4; i += 256) {
    const float4 u = hr[i];
    xr[i] = f16x4{norm_to_f16(u.x, r), norm_to_f16(u.y, r), norm_to_f16(u.z, r), norm_to_f16(u.w, r)};
  }
}

constexpr int ROPE_ROWS = 16;   // rows of R_l per block

// Rotate-half RoPE on the nq query heads and nkv key heads of ROPE_ROWS rows;
// q goes to q_out (f16).  Rows with kv_off >= 0 write their K (f16,
// token-major) at slab + kv_off and their V (f16) into the slot's V^T part
// (dimension-major: V^T[d][p % C] at slot + C*dkv*2 + (d*C + p % C)*2).  The
// V values are staged in LDS; a group of 8 rows that are 8 consecutive
// positions from a multiple of 8, all written to one slot, leaves as one
// 16-byte store per dimension, any other row as 2-byte stores.  Blocks are
// renumbered so that the row blocks one XCD runs at a time are adjacent and
// their partial V^T lines meet in that XCD's L2.
__global__ __launch_bounds__(256) void rope_kv_kernel(const float* __restrict__ qkv, int qkv_stride,
                                                      int M, const int32_t* __restrict__ pos,
                                                      const int64_t* __restrict__ kv_off,
                                                      const float2* __restrict__ cs, int nq,
                                                      int nkv, int hd, int C,
                                                      _Float16* __restrict__ q_out,
                                                      uint8_t* __restrict__ slab) {
  extern __shared__ _Float16 vstage[];     // [ROPE_ROWS][dkv]
  __shared__ int s_pos[ROPE_ROWS];         // position of the row
  __shared__ int s_pc[ROPE_ROWS];          // p % C, or -1 when the row writes no KV
  __shared__ int64_t s_k[ROPE_ROWS];       // byte offset of the row's K
  __shared__ int64_t s_vt[ROPE_ROWS];      // byte offset of V^T[0][p % C]
  __shared__ int s_fast[ROPE_ROWS / 8];
  const int nb = gridDim.x, b = blockIdx.x, per = nb / 8;
  const int blk = b < per * 8 ? (b % 8) * per + b / 8 : b;
  const int row0 = blk * ROPE_ROWS;
  const int nrows = min(ROPE_ROWS, M - row0);
  const int halfd = hd / 2, hq = hd / 8;   // quads per half head
  const int dq = nq * hd, dkv = nkv * hd;
  if (threadIdx.x < ROPE_ROWS) {
    const int row = row0 + threadIdx.x;
    const int64_t off = row < M && kv_off ? kv_off[row] : -1;
    const int p = row < M ? pos[row] : 0;
    const int pc = off >= 0 ? (p & (C - 1)) : -1;
    s_pos[threadIdx.x] = p;
    s_pc[threadIdx.x] = pc;
    s_k[threadIdx.x] = off;
    s_vt[threadIdx.x] = off >= 0 ? off - (int64_t)pc * dkv * 2 + (int64_t)C * dkv * 2 + pc * 2 : 0;
  }
  __syncthreads();
  // rotate 4 pairs (i..i+3, i+hd/2..i+hd/2+3) per item: float4 loads, 8-byte stores
  typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
  const int n_quads = (nq + nkv) * hq;
#pragma unroll 4
  for (int idx = threadIdx.x; idx < nrows * n_quads; idx += blockDim.x) {
    const int rr = idx / n_quads, qd = idx - rr * n_quads;
    const int head = qd / hq, i = (qd - head * hq) * 4;
    const float* x = qkv + (size_t)(row0 + rr) * qkv_stride + head * hd;  // q then k heads
    const float4 x1 = *reinterpret_cast<const float4*>(x + i);
    const float4 x2 = *reinterpret_cast<const float4*>(x + i + halfd);
    const float4* c = reinterpret_cast<const float4*>(cs + (size_t)s_pos[rr] * halfd + i);
    const float4 c01 = c[0], c23 = c[1];   // (cos, sin) of pairs i, i+1 and i+2, i+3
    const float2 r0 = rope_rotate(x1.x, x2.x, c01.x, c01.y), r1 = rope_rotate(x1.y, x2.y, c01.z, c01.w);
    const float2 r2 = rope_rotate(x1.z, x2.z, c23.x, c23.y), r3 = rope_rotate(x1.w, x2.w, c23.z, c23.w);
    const f16x4 y1 = {(_Float16)r0.x, (_Float16)r1.x, (_Float16)r2.x, (_Float16)r3.x};
    const f16x4 y2 = {(_Float16)r0.y, (_Float16)r1.y, (_Float16)r2.y, (_Float16)r3.y};
    _Float16* dst;
    if (head < nq) {
      dst = q_out + (size_t)(row0 + rr) * dq + head * hd;
    } else {
      if (s_pc[rr] < 0) continue;
      dst = reinterpret_cast<_Float16*>(slab + s_k[rr]) + (head - nq) * hd;
    }
    *reinterpret_cast<f16x4*>(dst + i) = y1;
    *reinterpret_cast<f16x4*>(dst + i + halfd) = y2;
  }
  const int vq = dkv / 4;
#pragma unroll 4
  for (int idx = threadIdx.x; idx < nrows * vq; idx += blockDim.x) {
    const int rr = idx / vq, d = (idx - rr * vq) * 4;
    const float4 v = *reinterpret_cast<const float4*>(qkv + (size_t)(row0 + rr) * qkv_stride + dq + dkv + d);
    *reinterpret_cast<f16x4*>(&vstage[rr * dkv + d]) = f16x4{(_Float16)v.x, (_Float16)v.y, (_Float16)v.z, (_Float16)v.w};
  }
  __syncthreads();
  if (threadIdx.x < ROPE_ROWS / 8) {
    const int g0 = threadIdx.x * 8;
    bool fast = s_pc[g0] >= 0 && (s_pc[g0] & 7) == 0;
    for (int i = 1; i < 8 && fast; ++i)
      fast = s_pc[g0 + i] == s_pc[g0] + i && s_vt[g0 + i] == s_vt[g0] + 2 * i;
    s_fast[threadIdx.x] = fast;
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < (ROPE_ROWS / 8) * dkv; idx += blockDim.x) {
    const int g = idx / dkv, d = idx % dkv, g0 = g * 8;
    if (s_fast[g]) {
      typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
      f16x8 v;
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = vstage[(g0 + i) * dkv + d];
      *reinterpret_cast<f16x8*>(slab + s_vt[g0] + (int64_t)d * C * 2) = v;
    } else {
      for (int i = 0; i < 8; ++i)
        if (s_pc[g0 + i] >= 0)
          *reinterpret_cast<_Float16*>(slab + s_vt[g0 + i] + (int64_t)d * C * 2) = vstage[(g0 + i) * dkv + d];
    }
  }
}

// One block per row: thread b dequantizes block b of the row.
// last_tok (device, or null): the last row's token, read from device memory
// instead of tok (a decode step whose token the previous step chose).
__global__ __launch_bounds__(256) void embed_kernel(const uint8_t* __restrict__ nib,
                                                    const uint16_t* __restrict__ scale,
                                                    const int32_t* __restrict__ tok, int d,
                                                    float* __restrict__ h, const int32_t* __restrict__ last_tok) {
  const int row = blockIdx.x;
  const int64_t t = (last_tok && row == (int)gridDim.x - 1) ? *last_tok : tok[row];
  const int nb = d / 32;
  float* out = h + (size_t)row * d;
  for (int b = threadIdx.x; b < nb; b += blockDim.x) {
    const uint4 q = *reinterpret_cast<const uint4*>(nib + t * (d / 2) + b * 16);
    const float dd = (float)__builtin_bit_cast(_Float16, scale[t * nb + b]);
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const uint32_t byte = (w[i] >> (8 * k)) & 0xFFu;
        out[b * 32 + 4 * i + k] = dd * (float)((int)(byte & 15u) - 8);
        out[b * 32 + 16 + 4 * i + k] = dd * (float)((int)(byte >> 4) - 8);
      }
  }
}

__global__ __launch_bounds__(256) void gather_rows_kernel(const float* __restrict__ src,
                                                          const int32_t* __restrict__ idx, int d,
                                                          float* __restrict__ dst) {
  const int row = blockIdx.x;
  const float4* s = reinterpret_cast<const float4*>(src + (size_t)idx[row] * d);
  float4* t = reinterpret_cast<float4*>(dst + (size_t)row * d);
  for (int i = threadIdx.x; i < d / 4; i += 256) t[i] = s[i];
}

constexpr int LM_ROWS = 256;   // vocabulary rows per block (64 per wave)
constexpr int LM_GROUP = 4;    // rows whose codes are in flight together per wave

// logits[v] = x . W_lm[v] with x = RMSNorm(h_last); per-block (max, lowest
// index) partials.  Lane l of every wave owns the 32-element blocks b = l,
// l + 64, ... of a row (NBL of them): their x values live in its registers
// (read once from global memory), so the row loop touches no LDS.  With
// codes q in 0..15, x . d (q - 8) over a block = d (sum x q - 8 sum x), the
// block's sum of x being precomputed; nibbles become floats with the
// byte-to-float conversions.  A wave takes its 64 rows LM_GROUP at a time,
// with two groups in flight: the loads of the next group are issued before
// the current one is summed.
// byte K of v as a float (one v_cvt_f32_ubyteK)
template <int K>
__device__ __forceinline__ float ubyte_f32(uint32_t v) { return (float)((v >> (8 * K)) & 0xFFu); }

template <int NBL>
__global__ __launch_bounds__(256) void lm_head_kernel(const float* __restrict__ h_last, int d,
                                                      float eps, const uint8_t* __restrict__ nib,
                                                      const uint16_t* __restrict__ scale,
                                                      int vocab, float* __restrict__ logits,
                                                      float* __restrict__ part_val,
                                                      int32_t* __restrict__ part_idx) {
  __shared__ float red[4];
  __shared__ float bval[4];
  __shared__ int32_t bidx[4];
  float ss = 0.f;
  for (int i = threadIdx.x; i < d; i += 256) {
    const float v = h_last[i];
    ss += v * v;
  }
  ss = block_sum256(ss, red);
  const float rn = 1.0f / __builtin_sqrtf(ss / (float)d + eps);

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int nb = d / 32;
  // this lane's blocks: x (normalised) and the sums of x over the low-nibble
  // half (elements 0..15) and the high-nibble half (16..31)
  float xv[NBL][32];
  float sx[NBL];
#pragma unroll
  for (int j = 0; j < NBL; ++j) {
    const int b = lane + 64 * j;
    sx[j] = 0.f;
#pragma unroll
    for (int e = 0; e < 32; e += 4) {
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (b < nb) v = *reinterpret_cast<const float4*>(h_last + b * 32 + e);
      xv[j][e] = v.x * rn;
      xv[j][e + 1] = v.y * rn;
      xv[j][e + 2] = v.z * rn;
      xv[j][e + 3] = v.w * rn;
      sx[j] += xv[j][e] + xv[j][e + 1] + xv[j][e + 2] + xv[j][e + 3];
    }
  }
  float best = -INFINITY;
  int32_t best_i = 0x7fffffff;
  const int v0 = blockIdx.x * LM_ROWS + w * (LM_ROWS / 4);
  // codes and scales of rows g .. g + LM_GROUP - 1 of this wave, from indices
  // clamped into range (blocks past the row's end read its last block and
  // meet x = 0; rows past the vocabulary read its last row and are not kept)
  auto load_group = [&](int g, uint4 (&q)[LM_GROUP][NBL], uint16_t (&sc)[LM_GROUP][NBL]) {
#pragma unroll
    for (int k = 0; k < LM_GROUP; ++k) {
      const int v = min(v0 + g + k, vocab - 1);
#pragma unroll
      for (int j = 0; j < NBL; ++j) {
        const int b = min(lane + 64 * j, nb - 1);
        q[k][j] = *reinterpret_cast<const uint4*>(nib + (int64_t)v * (d / 2) + b * 16);
        sc[k][j] = scale[(int64_t)v * nb + b];
      }
    }
  };
  auto dot_group = [&](int g, const uint4 (&q)[LM_GROUP][NBL], const uint16_t (&sc)[LM_GROUP][NBL]) {
#pragma unroll
    for (int k = 0; k < LM_GROUP; ++k) {
      float acc = 0.f;
#pragma unroll
      for (int j = 0; j < NBL; ++j) {
        const uint32_t wd[4] = {q[k][j].x, q[k][j].y, q[k][j].z, q[k][j].w};
        float dot = 0.f;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const uint32_t lo = wd[i] & 0x0F0F0F0Fu, hi = (wd[i] >> 4) & 0x0F0F0F0Fu;
          // byte kk of dword i: low nibble -> element 4i+kk, high -> 16+4i+kk
          dot = __builtin_fmaf(xv[j][4 * i + 0], ubyte_f32<0>(lo), dot);
          dot = __builtin_fmaf(xv[j][4 * i + 1], ubyte_f32<1>(lo), dot);
          dot = __builtin_fmaf(xv[j][4 * i + 2], ubyte_f32<2>(lo), dot);
          dot = __builtin_fmaf(xv[j][4 * i + 3], ubyte_f32<3>(lo), dot);
          dot = __builtin_fmaf(xv[j][16 + 4 * i + 0], ubyte_f32<0>(hi), dot);
          dot = __builtin_fmaf(xv[j][16 + 4 * i + 1], ubyte_f32<1>(hi), dot);
          dot = __builtin_fmaf(xv[j][16 + 4 * i + 2], ubyte_f32<2>(hi), dot);
          dot = __builtin_fmaf(xv[j][16 + 4 * i + 3], ubyte_f32<3>(hi), dot);
        }
        const float dd = (float)__builtin_bit_cast(_Float16, sc[k][j]);
        acc = __builtin_fmaf(dd, __builtin_fmaf(-8.0f, sx[j], dot), acc);
      }
      acc = wave_sum(acc);
      const int v = v0 + g + k;
      if (v < vocab) {
        if (acc > best) {   // rows ascend, so the first maximum keeps the lowest index
          best = acc;
          best_i = v;
        }
        if (lane == 0) logits[v] = acc;
      }
    }
  };
  // two groups in flight: the next group's codes load while this one is summed
  static_assert((LM_ROWS / 4) % (2 * LM_GROUP) == 0, "whole group pairs per wave");
  uint4 qa[LM_GROUP][NBL], qb[LM_GROUP][NBL];
  uint16_t sa[LM_GROUP][NBL], sb[LM_GROUP][NBL];
  load_group(0, qa, sa);
  for (int g = 0; g < LM_ROWS / 4; g += 2 * LM_GROUP) {
    load_group(g + LM_GROUP, qb, sb);
    dot_group(g, qa, sa);
    if (g + 2 * LM_GROUP < LM_ROWS / 4) load_group(g + 2 * LM_GROUP, qa, sa);
    dot_group(g + LM_GROUP, qb, sb);
  }
  if (lane == 0) {
    bval[w] = best;
    bidx[w] = best_i;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float bv = bval[0];
    int32_t bi = bidx[0];
    for (int i = 1; i < 4; ++i)
      if (bval[i] > bv || (bval[i] == bv && bidx[i] < bi)) {
        bv = bval[i];
        bi = bidx[i];
      }
    part_val[blockIdx.x] = bv;
    part_idx[blockIdx.x] = bi;
  }
}

__global__ __launch_bounds__(256) void argmax_kernel(const float* __restrict__ val,
                                                     const int32_t* __restrict__ idx, int n,
                                                     int32_t* __restrict__ token, int32_t* __restrict__ token2) {
  __shared__ float sv[256];
  __shared__ int32_t si[256];
  float bv = -INFINITY;
  int32_t bi = 0x7fffffff;
  for (int i = threadIdx.x; i < n; i += 256)
    if (val[i] > bv || (val[i] == bv && idx[i] < bi)) {
      bv = val[i];
      bi = idx[i];
    }
  sv[threadIdx.x] = bv;
  si[threadIdx.x] = bi;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if (threadIdx.x < s) {
      const float ov = sv[threadIdx.x + s];
      const int32_t oi = si[threadIdx.x + s];
      if (ov > sv[threadIdx.x] || (ov == sv[threadIdx.x] && oi < si[threadIdx.x])) {
        sv[threadIdx.x] = ov;
        si[threadIdx.x] = oi;
      }
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    *token = si[0];
    if (token2) *token2 = si[0];
  }
}

__global__ void fill_kernel(uint32_t* __restrict__ p, int64_t n, uint32_t value) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = value;
}

// wall_clock64() ticks at a constant 100 MHz on this target.
__global__ void spin_kernel(int64_t ticks) {
  const int64_t t0 = wall_clock64();
  for (int64_t it = 0; it < ticks + 1000; ++it) {   // each pass sleeps, so this bounds the wait
    if (wall_clock64() - t0 >= ticks) break;
    __builtin_amdgcn_s_sleep(8);
  }
}

}  // namespace

void launch_rmsnorm(const float* h, int m, int d, float eps, void* x, hipStream_t s) {
  hipLaunchKernelGGL(rmsnorm_kernel, dim3(m), dim3(256), 0, s, h, d, eps,
                     reinterpret_cast<_Float16*>(x));
}

void launch_rope_kv(const float* qkv, int qkv_stride, int m, const int32_t* pos,
                    const int64_t* kv_off, const float2* rope_cs, int nq, int nkv, int hd, int C,
                    void* q_out, void* slab, hipStream_t s) {
  const size_t lds = (size_t)ROPE_ROWS * nkv * hd * sizeof(_Float16);
  hipLaunchKernelGGL(rope_kv_kernel, dim3((m + ROPE_ROWS - 1) / ROPE_ROWS), dim3(256), lds, s, qkv,
                     qkv_stride, m, pos, kv_off, rope_cs, nq, nkv, hd, C,
                     reinterpret_cast<_Float16*>(q_out), reinterpret_cast<uint8_t*>(slab));
}

void launch_embed(const uint8_t* e_nib, const uint16_t* e_scale, const int32_t* tok, int m, int d,
                  float* h, hipStream_t s, const int32_t* last_tok) {
  hipLaunchKernelGGL(embed_kernel, dim3(m), dim3(256), 0, s, e_nib, e_scale, tok, d, h, last_tok);
}

void launch_gather_rows(const float* src, const int32_t* idx, int m, int d, float* dst,
                        hipStream_t s) {
  hipLaunchKernelGGL(gather_rows_kernel, dim3(m), dim3(256), 0, s, src, idx, d, dst);
}

void launch_lm_head(const float* h_last, int d, float eps, const uint8_t* w_nib,
                    const uint16_t* w_scale, int vocab, float* logits, float* part_val,
                    int32_t* part_idx, int32_t* token, hipStream_t s, int32_t* token2) {
  const int nblk = (vocab + LM_ROWS - 1) / LM_ROWS;
  const int nbl = (d / 32 + 63) / 64;   // 32-element blocks per lane (d <= 8192)
  switch (nbl) {
    case 1: hipLaunchKernelGGL(lm_head_kernel<1>, dim3(nblk), dim3(256), 0, s, h_last, d, eps, w_nib, w_scale,
                               vocab, logits, part_val, part_idx); break;
    case 2: hipLaunchKernelGGL(lm_head_kernel<2>, dim3(nblk), dim3(256), 0, s, h_last, d, eps, w_nib, w_scale,
                               vocab, logits, part_val, part_idx); break;
    case 3: hipLaunchKernelGGL(lm_head_kernel<3>, dim3(nblk), dim3(256), 0, s, h_last, d, eps, w_nib, w_scale,
                               vocab, logits, part_val, part_idx); break;
    default: hipLaunchKernelGGL(lm_head_kernel<4>, dim3(nblk), dim3(256), 0, s, h_last, d, eps, w_nib, w_scale,
                                vocab, logits, part_val, part_idx); break;
  }
  hipLaunchKernelGGL(argmax_kernel, dim3(1), dim3(256), 0, s, part_val, part_idx, nblk, token, token2);
}

void launch_fill(void* p, int64_t n_words, uint32_t value, hipStream_t s) {
  int64_t blocks = (n_words + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(fill_kernel, dim3((unsigned)blocks), dim3(256), 0, s,
                     reinterpret_cast<uint32_t*>(p), n_words, value);
}

void launch_zero(void* p, int64_t n_words, hipStream_t s) { launch_fill(p, n_words, 0u, s); }

void launch_spin(int64_t us, hipStream_t s) {
  if (us > 10000000) us = 10000000;
  hipLaunchKernelGGL(spin_kernel, dim3(1), dim3(64), 0, s, us * 100);
}

}  // namespace mzk
