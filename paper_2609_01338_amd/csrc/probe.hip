// Achievable ceilings of this GPU, measured rather than quoted: a dense f16
// MFMA stream whose operand bits keep changing (as real activations and
// weights do -- the clock of a power-limited chip depends on it), a plain
// device copy, and pinned host <-> device copies.  Used by the benchmark to
// state each kernel's rate against what the chip sustains next to the
// nominal peaks.
#include "mz_kernels.h"

namespace mzk {
namespace {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Each wave: iters x 16 v_mfma_f32_16x16x32_f16 on 16 independent
// accumulators; every 4 MFMAs one dword of each operand gets new bits (two
// multiply-adds and two masks per 64 MFMA cycles, so the VALU stays far from
// limiting).  Magnitudes stay below 2 (exponent field masked), so the fp32
// sums stay finite.
//
// MODE kProbeRandom: both operands random halves (dequantized weights and
// activations look like this).  MODE kProbeCodes: the B operand holds 4-bit
// codes q - 8 as exact halves (the weights of an exact-integer-weight GEMM;
// few mantissa bits toggle).  MODE kProbeBlockScaled: B as in kProbeCodes,
// each MFMA sums one 32-deep block into a zero accumulator and the block's
// fp32 scale is applied by four v_fma_f32 into the running sum (the whole
// per-MFMA cost of applying a Q4_0 block scale after the product).
enum { kProbeRandom = 0, kProbeCodes = 1, kProbeBlockScaled = 2 };

template <int MODE>
__global__ __launch_bounds__(512) void mfma_probe_kernel(float* __restrict__ out, int iters) {
  uint32_t s = threadIdx.x * 2654435761u + blockIdx.x * 40503u + 1u;
  u32x4 ra, rb;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    s = s * 1664525u + 1013904223u;
    ra[i] = (s & 0x3BFF3BFFu) ^ (0x80008000u * (s >> 31));
    s = s * 1664525u + 1013904223u;
    rb[i] = s & 0x3BFF3BFFu;
  }
  // two 4-bit codes -> halves 1024 + q (exponent with ulp 1) -> q - 8 exactly
  const f16x2 bias = {(_Float16)1032.0f, (_Float16)1032.0f};
  auto codes = [&](uint32_t x) {
    const f16x2 v = __builtin_bit_cast(f16x2, (x & 0x000F000Fu) | 0x64006400u) - bias;
    return __builtin_bit_cast(uint32_t, v);
  };
  u32x4 cb = rb;
  if (MODE != kProbeRandom) {
#pragma unroll
    for (int i = 0; i < 4; ++i) rb[i] = codes(cb[i]);
  }
  const float dsc = 1.0f + 1e-3f * (float)(threadIdx.x & 7);
  f32x4 acc[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int it = 0; it < iters; ++it) {
    f16x8 a = __builtin_bit_cast(f16x8, ra), b = __builtin_bit_cast(f16x8, rb);
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      if (MODE == kProbeBlockScaled) {
        asm volatile("" : "+v"(a));   // a distinct product each time (no reuse of an equal MFMA)
        const f32x4 t = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, f32x4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[i][r] = __builtin_fmaf(dsc, t[r], acc[i][r]);
      } else {
        acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, acc[i], 0, 0, 0);
      }
      if ((i & 3) == 3) {
        const int k = i >> 2;
        ra[k] = (ra[k] * 1664525u + 1013904223u) & 0xBBFFBBFFu;
        cb[k] = cb[k] * 22695477u + 1u;
        rb[k] = MODE == kProbeRandom ? (cb[k] & 0x3BFF3BFFu) : codes(cb[k] >> 7);
        a = __builtin_bit_cast(f16x8, ra);
        b = __builtin_bit_cast(f16x8, rb);
      }
    }
  }
  float t = 0.f;
#pragma unroll
  for (int i = 0; i < 16; ++i) t += acc[i][0] + acc[i][3];
  out[(size_t)blockIdx.x * blockDim.x + threadIdx.x] = t;
}

__global__ __launch_bounds__(256) void copy_probe_kernel(const uint4* __restrict__ src, uint4* __restrict__ dst,
                                                         int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) dst[i] = src[i];
}

}  // namespace

double mfma_probe_flops_per_launch(int blocks, int iters) {
  return (double)blocks * 8 * iters * 16 * (16.0 * 16 * 32 * 2);
}

void launch_mfma_probe(float* out, int blocks, int iters, int mode, hipStream_t s) {
  if (mode == kProbeCodes)
    hipLaunchKernelGGL(mfma_probe_kernel<kProbeCodes>, dim3(blocks), dim3(512), 0, s, out, iters);
  else if (mode == kProbeBlockScaled)
    hipLaunchKernelGGL(mfma_probe_kernel<kProbeBlockScaled>, dim3(blocks), dim3(512), 0, s, out, iters);
  else
    hipLaunchKernelGGL(mfma_probe_kernel<kProbeRandom>, dim3(blocks), dim3(512), 0, s, out, iters);
}

void launch_copy_probe(const void* src, void* dst, int64_t bytes, hipStream_t s) {
  hipLaunchKernelGGL(copy_probe_kernel, dim3(4096), dim3(256), 0, s, reinterpret_cast<const uint4*>(src),
                     reinterpret_cast<uint4*>(dst), bytes / 16);
}

}  // namespace mzk
