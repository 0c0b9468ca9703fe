// Memory-bound kernels of the restore-and-prefill path (gfx950): RMSNorm,
// rotary embedding with KV scatter into chunk slots, embedding gather with
// Q4_0 dequantization, row compaction, and the output head with argmax.
#include "mz_kernels.h"

namespace mzk {
namespace {

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Sum over a 256-thread block; every thread gets the result.
__device__ __forceinline__ float block_sum256(float v, float* red) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  return red[0] + red[1] + red[2] + red[3];
}

// One 256-thread block per row; d % 4 == 0.
__global__ __launch_bounds__(256) void rmsnorm_kernel(const float* __restrict__ h, int d, float eps,
                                                      _Float16* __restrict__ x) {
  __shared__ float red[4];
  const int row = blockIdx.x;
  const float4* hr = reinterpret_cast<const float4*>(h + (size_t)row * d);
  float ss = 0.f;
  for (int i = threadIdx.x; i < d / 4; i += 256) {
    const float4 v = hr[i];
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  ss = block_sum256(ss, red);
  const float r = 1.0f / __builtin_sqrtf(ss / (float)d + eps);
  typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
  f16x4* xr = reinterpret_cast<f16x4*>(x + (size_t)row * d);
  for (int i = threadIdx.x; i < d / 4; i += 256) {
    const float4 v = hr[i];
    xr[i] = f16x4{(_Float16)(v.x * r), (_Float16)(v.y * r), (_Float16)(v.z * r), (_Float16)(v.w * r)};
  }
}

// One block per row.  Rotate-half RoPE on the nq query heads and nkv key heads;
// q goes to q_out (f16), k and v to the row's slot (f16) when kv_off >= 0.
__global__ __launch_bounds__(256) void rope_kv_kernel(const float* __restrict__ qkv, int qkv_stride,
                                                      const int32_t* __restrict__ pos,
                                                      const int64_t* __restrict__ kv_off,
                                                      const float2* __restrict__ cs, int nq,
                                                      int nkv, int hd, int64_t v_delta,
                                                      _Float16* __restrict__ q_out,
                                                      uint8_t* __restrict__ slab) {
  const int row = blockIdx.x;
  const int halfd = hd / 2;
  const int dq = nq * hd, dkv = nkv * hd;
  const float* src = qkv + (size_t)row * qkv_stride;
  const int p = pos[row];
  const int64_t off = kv_off[row];
  const float2* c = cs + (size_t)p * halfd;
  _Float16* qo = q_out + (size_t)row * dq;
  _Float16* ko = off >= 0 ? reinterpret_cast<_Float16*>(slab + off) : nullptr;
  const int n_pairs = (nq + nkv) * halfd;
  for (int idx = threadIdx.x; idx < n_pairs; idx += blockDim.x) {
    const int head = idx / halfd, i = idx % halfd;
    const float2 t = c[i];
    const float* x = src + head * hd;   // q heads then k heads are contiguous
    const float x1 = x[i], x2 = x[i + halfd];
    const float y1 = x1 * t.x - x2 * t.y;
    const float y2 = x2 * t.x + x1 * t.y;
    if (head < nq) {
      qo[head * hd + i] = (_Float16)y1;
      qo[head * hd + i + halfd] = (_Float16)y2;
    } else if (ko) {
      const int g = head - nq;
      ko[g * hd + i] = (_Float16)y1;
      ko[g * hd + i + halfd] = (_Float16)y2;
    }
  }
  if (ko) {
    _Float16* vo = reinterpret_cast<_Float16*>(slab + off + v_delta);
    const float* v = src + dq + dkv;
    for (int i = threadIdx.x; i < dkv; i += blockDim.x) vo[i] = (_Float16)v[i];
  }
}

// One block per row: thread b dequantizes block b of the row.
__global__ __launch_bounds__(256) void embed_kernel(const uint8_t* __restrict__ nib,
                                                    const uint16_t* __restrict__ scale,
                                                    const int32_t* __restrict__ tok, int d,
                                                    float* __restrict__ h) {
  const int row = blockIdx.x;
  const int64_t t = tok[row];
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

constexpr int LM_ROWS = 64;   // vocabulary rows per block (16 per wave)

// logits[v] = x . W_lm[v] with x = RMSNorm(h_last) staged in LDS; per-block
// (max, lowest index) partials.
__global__ __launch_bounds__(256) void lm_head_kernel(const float* __restrict__ h_last, int d,
                                                      float eps, const uint8_t* __restrict__ nib,
                                                      const uint16_t* __restrict__ scale,
                                                      int vocab, float* __restrict__ logits,
                                                      float* __restrict__ part_val,
                                                      int32_t* __restrict__ part_idx) {
  extern __shared__ float xs[];
  __shared__ float red[4];
  __shared__ float bval[4];
  __shared__ int32_t bidx[4];
  float ss = 0.f;
  for (int i = threadIdx.x; i < d; i += 256) {
    const float v = h_last[i];
    xs[i] = v;
    ss += v * v;
  }
  ss = block_sum256(ss, red);
  const float r = 1.0f / __builtin_sqrtf(ss / (float)d + eps);
  for (int i = threadIdx.x; i < d; i += 256) xs[i] *= r;
  __syncthreads();

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int nb = d / 32;
  float best = -INFINITY;
  int32_t best_i = 0x7fffffff;
  for (int k = 0; k < LM_ROWS / 4; ++k) {
    const int v = blockIdx.x * LM_ROWS + w * (LM_ROWS / 4) + k;
    if (v >= vocab) break;
    float acc = 0.f;
    for (int b = lane; b < nb; b += 64) {
      const uint4 q = *reinterpret_cast<const uint4*>(nib + (int64_t)v * (d / 2) + b * 16);
      const float dd = (float)__builtin_bit_cast(_Float16, scale[(int64_t)v * nb + b]);
      const uint32_t wd[4] = {q.x, q.y, q.z, q.w};
      const float* xb = xs + b * 32;
      float sl = 0.f, sh = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
          const uint32_t byte = (wd[i] >> (8 * kk)) & 0xFFu;
          sl += xb[4 * i + kk] * (float)((int)(byte & 15u) - 8);
          sh += xb[16 + 4 * i + kk] * (float)((int)(byte >> 4) - 8);
        }
      acc += dd * (sl + sh);
    }
    acc = wave_sum(acc);
    if (acc > best) {   // rows ascend, so the first maximum keeps the lowest index
      best = acc;
      best_i = v;
    }
    if (lane == 0) logits[v] = acc;
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
                                                     int32_t* __restrict__ token) {
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
  if (threadIdx.x == 0) *token = si[0];
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
                    const int64_t* kv_off, const float2* rope_cs, int nq, int nkv, int hd,
                    int64_t v_delta, void* q_out, void* slab, hipStream_t s) {
  hipLaunchKernelGGL(rope_kv_kernel, dim3(m), dim3(256), 0, s, qkv, qkv_stride, pos, kv_off, rope_cs, nq, nkv,
                     hd, v_delta, reinterpret_cast<_Float16*>(q_out),
                     reinterpret_cast<uint8_t*>(slab));
}

void launch_embed(const uint8_t* e_nib, const uint16_t* e_scale, const int32_t* tok, int m, int d,
                  float* h, hipStream_t s) {
  hipLaunchKernelGGL(embed_kernel, dim3(m), dim3(256), 0, s, e_nib, e_scale, tok, d, h);
}

void launch_gather_rows(const float* src, const int32_t* idx, int m, int d, float* dst,
                        hipStream_t s) {
  hipLaunchKernelGGL(gather_rows_kernel, dim3(m), dim3(256), 0, s, src, idx, d, dst);
}

void launch_lm_head(const float* h_last, int d, float eps, const uint8_t* w_nib,
                    const uint16_t* w_scale, int vocab, float* logits, float* part_val,
                    int32_t* part_idx, int32_t* token, hipStream_t s) {
  const int nblk = (vocab + LM_ROWS - 1) / LM_ROWS;
  hipLaunchKernelGGL(lm_head_kernel, dim3(nblk), dim3(256), d * sizeof(float), s, h_last, d, eps,
                     w_nib, w_scale, vocab, logits, part_val, part_idx);
  hipLaunchKernelGGL(argmax_kernel, dim3(1), dim3(256), 0, s, part_val, part_idx, nblk, token);
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
