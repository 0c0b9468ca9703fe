// Block-wide sums and the RMSNorm scale of one row, shared by the RMSNorm
// kernel and the single-row GEMV that normalizes its own input: both take
// the scale through this one routine, so the f16 values they form from it,
// (f16)(h * r), are the same bits.
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
    ss += v[k].x * v[k].x + v[k].y * v[k].y + v[k].z * v[k].z + v[k].w * v[k].w;
  }
  for (int i = threadIdx.x + kRowNormRegs * 256; i < n4; i += 256) {
    const float4 u = h4[i];
    ss += u.x * u.x + u.y * u.y + u.z * u.z + u.w * u.w;
  }
  ss = block_sum256(ss, red);
  return 1.0f / __builtin_sqrtf(ss / (float)d + eps);
}

}  // namespace mzk
