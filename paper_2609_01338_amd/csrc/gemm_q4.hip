// Q4_0-weight GEMM for gfx950: Y = X . W^T, X f16 [m][k], W Q4_0 [n][k].
//
// A 512-thread workgroup computes a 256 x 256 tile of Y.  Each 64-wide K step
// stages the activation tile (f16) and the weight tile in LDS (double
// buffered, one barrier a step); the weight tile arrives as Q4_0 (2 blocks of
// 32 per row: 16 nibble bytes + an fp16 scale each) and is dequantized on the
// way into LDS.  The nibbles are pre-ordered (at load time) so that one
// and-or per pair of codes builds two halves 1024 + q; a packed subtract of
// 1032 gives q - 8 exactly and a packed multiply by the scale gives
// d * (q - 8) rounded once to f16 (2^-11 relative).  Eight waves in a 4 x 2
// grid each own a 64 x 128 sub-tile as 4 x 8 tiles of v_mfma_f32_16x16x32_f16
// with fp32 accumulation.  (f16 rather than bf16 operands: same MFMA rate on
// this chip, three more mantissa bits, and the activations of this model stay
// far inside the f16 range.)
//
// Workgroups are numbered so that each XCD (workgroups are dealt to the 8 XCDs
// round-robin) walks a contiguous run of tiles, M-major: neighbouring tiles on
// one XCD share the activation rows in that XCD's L2.
//
// MFMA 16x16x32 operand layout (checked on gfx950): lane l feeds row/column
// l % 16 with the 8 consecutive k of group l / 16; the accumulator holds rows
// 4 * (l / 16) + r (r = 0..3) of column l % 16.
#include "mz_kernels.h"

namespace mzk {
namespace {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int BM = 256, BN = kGemmTileN, BK = kGemmTileK;
constexpr int NT = 512;                     // threads
constexpr int LDS_STRIDE = BK + 8;          // halves per LDS row: 144 B, conflict-free b128 reads
constexpr int NIB_BYTES = BN * BK / 2;      // 8192

__device__ __forceinline__ float silu(float g) { return g / (1.0f + __expf(-g)); }

__device__ __forceinline__ uint32_t pair_code(uint32_t w, int shift) {
  // two 4-bit codes at bits [shift, shift+4) and [16+shift, 20+shift) -> halves 1024 + q
  return ((w >> shift) & 0x000F000Fu) | 0x64006400u;
}

__device__ __forceinline__ uint32_t dequant_pair(uint32_t w, int shift, f16x2 d2) {
  const f16x2 c = __builtin_bit_cast(f16x2, pair_code(w, shift));
  const f16x2 off = {(_Float16)1032.0f, (_Float16)1032.0f};
  return __builtin_bit_cast(uint32_t, (c - off) * d2);
}

// One pre-ordered Q4_0 block (4 dwords; dword i holds elements 8i..8i+7) ->
// 32 halves in LDS.
__device__ __forceinline__ void dequant_block_to_lds(uint4 nib, uint16_t dbits, _Float16* dst) {
  const _Float16 d = __builtin_bit_cast(_Float16, dbits);
  const f16x2 d2 = {d, d};
  const uint32_t w[4] = {nib.x, nib.y, nib.z, nib.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint4 o;
    o.x = dequant_pair(w[i], 0, d2);
    o.y = dequant_pair(w[i], 4, d2);
    o.z = dequant_pair(w[i], 8, d2);
    o.w = dequant_pair(w[i], 12, d2);
    *reinterpret_cast<uint4*>(dst + 8 * i) = o;
  }
}

template <int EPI>
__global__ __launch_bounds__(NT) void gemm_q4_kernel(const _Float16* __restrict__ X, int M, int K,
                                                     const uint8_t* __restrict__ Wp, int N,
                                                     void* __restrict__ Y) {
  extern __shared__ __attribute__((aligned(16))) _Float16 lds[];
  _Float16* As = lds;                              // [2][BM * LDS_STRIDE]
  _Float16* Bs = lds + 2 * BM * LDS_STRIDE;        // [2][BN * LDS_STRIDE]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave & 3, wn = wave >> 2;
  const int n_tiles = N / BN;
  // XCD-contiguous tile order
  const int total = gridDim.x;
  const int b = blockIdx.x;
  const int per = total / 8;
  const int t = b < per * 8 ? (b % 8) * per + b / 8 : b;
  const int mt = t / n_tiles, nt = t % n_tiles;
  const int nk = K / BK;

  // activation loads: 4 segments of 16 B per thread (rows tid/8 + 64 i, column tid%8)
  const int a_row = tid >> 3, a_c16 = tid & 7;
  const _Float16* x0 = X + (size_t)min(mt * BM + a_row, M - 1) * K + a_c16 * 8;
  const _Float16* x1 = X + (size_t)min(mt * BM + a_row + 64, M - 1) * K + a_c16 * 8;
  const _Float16* x2 = X + (size_t)min(mt * BM + a_row + 128, M - 1) * K + a_c16 * 8;
  const _Float16* x3 = X + (size_t)min(mt * BM + a_row + 192, M - 1) * K + a_c16 * 8;
  const int a_lds = a_row * LDS_STRIDE + a_c16 * 8;
  // weight loads: one Q4_0 block (row tid/2, block tid%2) per thread
  const uint8_t* wtile = Wp + (size_t)nt * nk * kGemmTileBytes;
  const int b_lds = (tid >> 1) * LDS_STRIDE + (tid & 1) * 32;

  f32x4 acc[4][8];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  uint4 ra0, ra1, ra2, ra3, rnib;
  uint16_t rsc;
#define MZ_GLOAD(kt)                                                                    \
  do {                                                                                  \
    const int ko_ = (kt) * BK;                                                          \
    ra0 = *reinterpret_cast<const uint4*>(x0 + ko_);                                    \
    ra1 = *reinterpret_cast<const uint4*>(x1 + ko_);                                    \
    ra2 = *reinterpret_cast<const uint4*>(x2 + ko_);                                    \
    ra3 = *reinterpret_cast<const uint4*>(x3 + ko_);                                    \
    const uint8_t* t_ = wtile + (size_t)(kt) * kGemmTileBytes;                          \
    rnib = *reinterpret_cast<const uint4*>(t_ + tid * 16);                              \
    rsc = *reinterpret_cast<const uint16_t*>(t_ + NIB_BYTES + tid * 2);                 \
  } while (0)
#define MZ_LSTORE(st)                                                                   \
  do {                                                                                  \
    _Float16* a_ = As + (st) * BM * LDS_STRIDE + a_lds;                                 \
    *reinterpret_cast<uint4*>(a_) = ra0;                                                \
    *reinterpret_cast<uint4*>(a_ + 64 * LDS_STRIDE) = ra1;                              \
    *reinterpret_cast<uint4*>(a_ + 128 * LDS_STRIDE) = ra2;                             \
    *reinterpret_cast<uint4*>(a_ + 192 * LDS_STRIDE) = ra3;                             \
    dequant_block_to_lds(rnib, rsc, Bs + (st) * BN * LDS_STRIDE + b_lds);               \
  } while (0)

  MZ_GLOAD(0);
  MZ_LSTORE(0);
  __syncthreads();

  const int frag_row = lane & 15;
  const int frag_k = (lane >> 4) * 8;
  for (int kt = 0; kt < nk; ++kt) {
    const int st = kt & 1;
    if (kt + 1 < nk) MZ_GLOAD(kt + 1);
    const _Float16* Ab = As + st * BM * LDS_STRIDE + (wm * 64 + frag_row) * LDS_STRIDE + frag_k;
    const _Float16* Bb = Bs + st * BN * LDS_STRIDE + (wn * 128 + frag_row) * LDS_STRIDE + frag_k;
#pragma unroll
    for (int ks = 0; ks < BK / 32; ++ks) {
      f16x8 a[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        a[i] = *reinterpret_cast<const f16x8*>(Ab + i * 16 * LDS_STRIDE + ks * 32);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const f16x8 bf = *reinterpret_cast<const f16x8*>(Bb + j * 16 * LDS_STRIDE + ks * 32);
#pragma unroll
        for (int i = 0; i < 4; ++i)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a[i], bf, acc[i][j], 0, 0, 0);
      }
    }
    if (kt + 1 < nk) MZ_LSTORE(st ^ 1);
    __syncthreads();
  }
#undef MZ_GLOAD
#undef MZ_LSTORE

  // epilogue
  const int col_in = lane & 15;
  const int row_in = (lane >> 4) * 4;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = mt * BM + wm * 64 + i * 16 + row_in + r;
      if (row >= M) continue;
      if (EPI == kEpiSwiGLU) {
        _Float16* y = reinterpret_cast<_Float16*>(Y) + (size_t)row * (N / 2);
#pragma unroll
        for (int jp = 0; jp < 4; ++jp) {
          const float g = acc[i][2 * jp][r], u = acc[i][2 * jp + 1][r];
          const int col = nt * (BN / 2) + wn * 64 + jp * 16 + col_in;
          y[col] = (_Float16)(silu(g) * u);
        }
      } else {
        float* y = reinterpret_cast<float*>(Y) + (size_t)row * N;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int col = nt * BN + wn * 128 + j * 16 + col_in;
          if (EPI == kEpiAdd)
            y[col] += acc[i][j][r];
          else
            y[col] = acc[i][j][r];
        }
      }
    }
  }
}

constexpr size_t kLdsBytes = (size_t)2 * (BM + BN) * LDS_STRIDE * sizeof(_Float16);

}  // namespace

void launch_gemm_q4(const void* x, int m, int n, int k, const void* w, int epilogue, void* y,
                    hipStream_t s) {
  static const bool lds_ok = [] {   // allow more than 64 KB of dynamic LDS, once per process
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_q4_kernel<kEpiStore>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsBytes);
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_q4_kernel<kEpiAdd>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsBytes);
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_q4_kernel<kEpiSwiGLU>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsBytes);
    return true;
  }();
  (void)lds_ok;
  const int tiles = (n / BN) * ((m + BM - 1) / BM);
  const _Float16* X = reinterpret_cast<const _Float16*>(x);
  const uint8_t* W = reinterpret_cast<const uint8_t*>(w);
  switch (epilogue) {
    case kEpiStore:
      hipLaunchKernelGGL(gemm_q4_kernel<kEpiStore>, dim3(tiles), dim3(NT), kLdsBytes, s, X, m, k, W,
                         n, y);
      break;
    case kEpiAdd:
      hipLaunchKernelGGL(gemm_q4_kernel<kEpiAdd>, dim3(tiles), dim3(NT), kLdsBytes, s, X, m, k, W, n,
                         y);
      break;
    default:
      hipLaunchKernelGGL(gemm_q4_kernel<kEpiSwiGLU>, dim3(tiles), dim3(NT), kLdsBytes, s, X, m, k,
                         W, n, y);
      break;
  }
}

}  // namespace mzk
