// 8-bit group-wise codec of swapped KV chunks (the paper's default codec on
// its in-memory swap path, Sec. 5, after FlexGen's group-wise quantization).
//
// On a run of n halves (n a multiple of 64), groups of 64 consecutive values:
//   mn, mx = min, max (exact in fp32);  d = half(fp32(mx - mn) / 255);  m = mn
//   q_i = d == 0 ? 0 : clamp(rint(fp32(x_i - m) / fp32(d)), 0, 255)
//   x^_i = half(fp32(q_i) * fp32(d) + fp32(m))   (the product is exact)
// with correctly rounded fp32 division and round-half-even, so every code is
// reproducible bit for bit.  Compressed run: n code bytes, then (m, d) as two
// halves per group.  A wave takes four groups, 16 lanes per group, 4 values
// (8 bytes in, 4 code bytes out) per lane.
#include "mz_kernels.h"

namespace mzk {
namespace {

typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));

constexpr int G = 64;   // values per group

__device__ __forceinline__ float group16_min(float v) {
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) v = fminf(v, __shfl_xor(v, o, 16));
  return v;
}
__device__ __forceinline__ float group16_max(float v) {
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) v = fmaxf(v, __shfl_xor(v, o, 16));
  return v;
}

// blockIdx.y selects one of n_runs runs: run r reads src + src_off(r) and
// writes dst + r * (n + n/16) (compress) -- see the launchers.
__global__ __launch_bounds__(256) void kv_compress_kernel(const uint8_t* __restrict__ src_base,
                                                          const int32_t* __restrict__ src_slots,
                                                          int64_t src_stride, int64_t n,
                                                          uint8_t* __restrict__ dst) {
  const int64_t gid = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 4;   // group
  const int sub = threadIdx.x & 15;
  if (gid * G >= n) return;   // whole 16-lane groups leave together
  const int r = blockIdx.y;
  const _Float16* src = reinterpret_cast<const _Float16*>(
      src_base + (src_slots ? (int64_t)src_slots[r] : (int64_t)r) * src_stride);
  uint8_t* out = dst + (int64_t)r * (n + n / 16);
  const f16x4 v = *reinterpret_cast<const f16x4*>(src + gid * G + sub * 4);
  float x[4] = {(float)v[0], (float)v[1], (float)v[2], (float)v[3]};
  const float mn = group16_min(fminf(fminf(x[0], x[1]), fminf(x[2], x[3])));
  const float mx = group16_max(fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])));
  const _Float16 dh = (_Float16)__fdiv_rn(mx - mn, 255.0f);
  const float d = (float)dh;
  uint32_t packed = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float q = d == 0.0f ? 0.0f : __builtin_rintf(__fdiv_rn(x[i] - mn, d));
    q = fminf(fmaxf(q, 0.0f), 255.0f);
    packed |= (uint32_t)q << (8 * i);
  }
  *reinterpret_cast<uint32_t*>(out + gid * G + sub * 4) = packed;
  if (sub == 0) {
    const _Float16 p[2] = {(_Float16)mn, dh};
    *reinterpret_cast<uint32_t*>(out + n + gid * 4) = __builtin_bit_cast(uint32_t, p);
  }
}

__global__ __launch_bounds__(256) void kv_decompress_kernel(const uint8_t* __restrict__ src, int64_t n,
                                                            uint8_t* __restrict__ dst_base,
                                                            const int32_t* __restrict__ dst_slots,
                                                            int64_t dst_stride) {
  const int64_t lane4 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;   // 4 values each
  if (lane4 * 4 >= n) return;
  const int r = blockIdx.y;
  const uint8_t* in = src + (int64_t)r * (n + n / 16);
  _Float16* out = reinterpret_cast<_Float16*>(
      dst_base + (dst_slots ? (int64_t)dst_slots[r] : (int64_t)r) * dst_stride);
  const int64_t g = lane4 * 4 / G;
  const uint32_t codes = *reinterpret_cast<const uint32_t*>(in + lane4 * 4);
  const uint32_t pw = *reinterpret_cast<const uint32_t*>(in + n + g * 4);
  const float m = (float)__builtin_bit_cast(_Float16, (uint16_t)(pw & 0xFFFFu));
  const float d = (float)__builtin_bit_cast(_Float16, (uint16_t)(pw >> 16));
  f16x4 o;
#pragma unroll
  for (int i = 0; i < 4; ++i) o[i] = (_Float16)__builtin_fmaf((float)((codes >> (8 * i)) & 0xFFu), d, m);
  *reinterpret_cast<f16x4*>(out + lane4 * 4) = o;
}

}  // namespace

int64_t kv_compressed_bytes(int64_t n_halves) { return n_halves + n_halves / 16; }

void launch_kv_compress(const void* src_base, const int32_t* src_slots, int64_t src_stride, int64_t n_halves,
                        int n_runs, void* dst, hipStream_t s) {
  if (n_runs < 1 || n_halves < G) return;
  const int64_t threads = n_halves / G * 16;
  hipLaunchKernelGGL(kv_compress_kernel, dim3((unsigned)((threads + 255) / 256), n_runs), dim3(256), 0, s,
                     reinterpret_cast<const uint8_t*>(src_base), src_slots, src_stride, n_halves,
                     reinterpret_cast<uint8_t*>(dst));
}

void launch_kv_decompress(const void* src, int64_t n_halves, int n_runs, void* dst_base,
                          const int32_t* dst_slots, int64_t dst_stride, hipStream_t s) {
  if (n_runs < 1 || n_halves < G) return;
  const int64_t threads = n_halves / 4;
  hipLaunchKernelGGL(kv_decompress_kernel, dim3((unsigned)((threads + 255) / 256), n_runs), dim3(256), 0, s,
                     reinterpret_cast<const uint8_t*>(src), n_halves, reinterpret_cast<uint8_t*>(dst_base),
                     dst_slots, dst_stride);
}

}  // namespace mzk
