// The rotary-embedding rotation shared by every kernel that applies it: the
// query and key/value GEMM epilogues, the reduce of their split-K forms and
// the standalone RoPE pass.  Each output is one fused multiply-add onto a
// rounded product, written out so that no compiler contraction choice can
// differ between them: the fused and the separate paths give the same bits.
#pragma once
#include <hip/hip_runtime.h>

namespace mzk {

// Rotate-half pair (x1, x2) of one frequency by (c, s) = (cos, sin):
// (x1 c - x2 s, x2 c + x1 s), rounded to fp32.  The empty asm keeps the
// results in fp32 registers: a caller that converts them to f16 would
// otherwise let the compiler merge the multiply-add and the conversion into
// one mixed-precision instruction (a single rounding to f16) in some kernels
// and not in others.
__device__ __forceinline__ float2 rope_rotate(float x1, float x2, float c, float s) {
  float a = __builtin_fmaf(x1, c, -(x2 * s)), b = __builtin_fmaf(x2, c, x1 * s);
  asm volatile("" : "+v"(a), "+v"(b));
  return make_float2(a, b);
}

}  // namespace mzk
