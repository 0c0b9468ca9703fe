// Block-wide sums and the RMSNorm scale of one row, shared by the RMSNorm
// kernel and the single-row GEMV that normalizes its own input: both take
// the scale and form (f16)(h * r) through these routines, so their values
// are the same bits.
#pragma once
#include <hip/hip_runtime.h>

namespace mzk {

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

// acc + x.x^2 + x.y^2 + x.z^2 + x.w^2 as a chain of fused multiply-adds in
// that order (no contraction choice left to the compiler).
__device__ __forceinline__ float sumsq4(float4 x, float acc) {
  acc = __builtin_fmaf(x.x, x.x, acc);
  acc = __builtin_fmaf(x.y, x.y, acc);
  acc = __builtin_fmaf(x.z, x.z, acc);
  return __builtin_fmaf(x.w, x.w, acc);
}

// r = 1 / sqrt(mean(h^2) + eps) of the fp32 row hr (d elements, d % 4 == 0)
// by a 256-thread block (red: 4 floats of LDS).  Thread t sums the squares
// of float4 pieces t, t + 256, ...; the first kRowNormRegs of its pieces are
// left in v (zeros past the row) for a caller that scales them.
constexpr int kRowNormRegs = 8;
__device__ __forceinline__ float row_inv_rms(const float* __restrict__ hr, int d, float eps,
                                             float4 (&v)[kRowNormRegs], float* red) {
  const int n4 = d / 4;
  const float4* h4 = reinterpret_cast<const float4*>(hr);
  float ss = 0.f;
#pragma unroll
  for (int k = 0; k < kRowNormRegs; ++k) {
    const int i = threadIdx.x + k * 256;
    v[k] = i < n4 ? h4[i] : float4{0.f, 0.f, 0.f, 0.f};
    ss = sumsq4(v[k], ss);
  }
  for (int i = threadIdx.x + kRowNormRegs * 256; i < n4; i += 256) ss = sumsq4(h4[i], ss);
  ss = block_sum256(ss, red);
  return 1.0f / __builtin_sqrtf(ss / (float)d + eps);
}

// (f16)(h * r) for every producer of normalized activations: the product
// is rounded to fp32 and then to f16.  The empty asm keeps the compiler from
// merging the multiply and the conversion into one mixed-precision
// instruction (a single rounding) in some kernels and not in others.
__device__ __forceinline__ _Float16 norm_to_f16(float h, float r) {
  float p = h * r;
  asm volatile("" : "+v"(p));
  return (_Float16)p;
}

}  // namespace mzk
