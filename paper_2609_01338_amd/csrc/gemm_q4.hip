// Q4_0-weight GEMM for gfx950: Y = X . W^T, X f16 [m][k], W Q4_0 [n][k].
//
// A 256-thread workgroup computes a 128 x 128 tile of Y.  Each 64-wide K step
// stages the activation tile (f16) and the weight tile in LDS; the weight
// tile arrives as Q4_0 (2 blocks of 32 per row: 16 nibble bytes + an fp16
// scale each) and is dequantized on the way into LDS, w = d * (q - 8), which
// is exact in fp32 and then rounded to f16 (2^-11 relative).  Four waves in a
// 2 x 2 grid each own a 64 x 64 sub-tile as 4 x 4 tiles of
// v_mfma_f32_16x16x32_f16 with fp32 accumulation.  (f16 rather than bf16
// operands: same MFMA rate on this chip, three more mantissa bits, and the
// activations of this model stay far inside the f16 range.)  Global loads for
// step k+1 are issued before the MFMAs of step k and stored to the other LDS
// buffer after them (one barrier a step).
//
// MFMA 16x16x32 operand layout (checked on gfx950): lane l feeds row/column
// l % 16 with the 8 consecutive k of group l / 16; the accumulator holds rows
// 4 * (l / 16) + r (r = 0..3) of column l % 16.
#include "mz_kernels.h"

namespace mzk {
namespace {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int BM = 128, BN = kGemmTileN, BK = kGemmTileK;
constexpr int LDS_STRIDE = BK + 8;          // halves per LDS row: 144 B, conflict-free b128 reads
constexpr int NIB_BYTES = BN * BK / 2;      // 4096

__device__ __forceinline__ float silu(float g) { return g / (1.0f + __expf(-g)); }

// Dequantize one Q4_0 block (16 nibble bytes as 4 dwords, scale d) into
// 32 f16 at dst (element j in low nibble of byte j, j+16 in its high nibble).
__device__ __forceinline__ void dequant_block_to_lds(uint4 nib, float d, _Float16* dst) {
  const float m8 = -8.0f * d;
  uint32_t w[4] = {nib.x, nib.y, nib.z, nib.w};
  f16x8 v[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint32_t lo = w[i] & 0x0F0F0F0Fu;
    uint32_t hi = (w[i] >> 4) & 0x0F0F0F0Fu;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      float ql = (float)((lo >> (8 * b)) & 0xFFu);
      float qh = (float)((hi >> (8 * b)) & 0xFFu);
      // elements 4i+b (low) and 16+4i+b (high)
      v[(4 * i + b) >> 3][(4 * i + b) & 7] = (_Float16)__builtin_fmaf(ql, d, m8);
      v[(16 + 4 * i + b) >> 3][(16 + 4 * i + b) & 7] = (_Float16)__builtin_fmaf(qh, d, m8);
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) *reinterpret_cast<f16x8*>(dst + 8 * i) = v[i];
}

template <int EPI>
__global__ __launch_bounds__(256) void gemm_q4_kernel(const _Float16* __restrict__ X, int M, int K,
                                                      const uint8_t* __restrict__ Wp, int N,
                                                      void* __restrict__ Y) {
  __shared__ __attribute__((aligned(16))) _Float16 As[2][BM * LDS_STRIDE];
  __shared__ __attribute__((aligned(16))) _Float16 Bs[2][BN * LDS_STRIDE];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int nt = blockIdx.x;
  const int mt = blockIdx.y;
  const int nk = K / BK;

  // activation loads: 4 segments of 16 B per thread
  const _Float16* xrow[4];
  int a_lds[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int seg = tid + 256 * i;
    int row = seg >> 3, c16 = seg & 7;
    int gr = mt * BM + row;
    gr = gr < M ? gr : M - 1;
    xrow[i] = X + (size_t)gr * K + c16 * 8;
    a_lds[i] = row * LDS_STRIDE + c16 * 8;
  }
  // weight loads: one Q4_0 block (row tid/2, block tid%2) per thread
  const uint8_t* wtile = Wp + (size_t)nt * nk * kGemmTileBytes;
  const int b_lds = (tid >> 1) * LDS_STRIDE + (tid & 1) * 32;

  uint4 ra[4];
  uint4 rnib;
  uint16_t rsc;
  auto gload = [&](int kt) {
#pragma unroll
    for (int i = 0; i < 4; ++i) ra[i] = *reinterpret_cast<const uint4*>(xrow[i] + kt * BK);
    const uint8_t* t = wtile + (size_t)kt * kGemmTileBytes;
    rnib = *reinterpret_cast<const uint4*>(t + tid * 16);
    rsc = *reinterpret_cast<const uint16_t*>(t + NIB_BYTES + tid * 2);
  };
  auto lstore = [&](int st) {
#pragma unroll
    for (int i = 0; i < 4; ++i) *reinterpret_cast<uint4*>(&As[st][a_lds[i]]) = ra[i];
    float d = (float)__builtin_bit_cast(_Float16, rsc);
    dequant_block_to_lds(rnib, d, &Bs[st][b_lds]);
  };

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  gload(0);
  lstore(0);
  __syncthreads();

  const int frag_row = lane & 15;
  const int frag_k = (lane >> 4) * 8;
  for (int kt = 0; kt < nk; ++kt) {
    const int st = kt & 1;
    if (kt + 1 < nk) gload(kt + 1);
#pragma unroll
    for (int ks = 0; ks < BK / 32; ++ks) {
      f16x8 a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        a[i] = *reinterpret_cast<const f16x8*>(
            &As[st][(wm * 64 + i * 16 + frag_row) * LDS_STRIDE + ks * 32 + frag_k]);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        b[j] = *reinterpret_cast<const f16x8*>(
            &Bs[st][(wn * 64 + j * 16 + frag_row) * LDS_STRIDE + ks * 32 + frag_k]);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) lstore(st ^ 1);
    __syncthreads();
  }

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
        for (int jp = 0; jp < 2; ++jp) {
          const float g = acc[i][2 * jp][r], u = acc[i][2 * jp + 1][r];
          const int col = nt * (BN / 2) + wn * 32 + jp * 16 + col_in;
          y[col] = (_Float16)(silu(g) * u);
        }
      } else {
        float* y = reinterpret_cast<float*>(Y) + (size_t)row * N;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int col = nt * BN + wn * 64 + j * 16 + col_in;
          if (EPI == kEpiAdd)
            y[col] += acc[i][j][r];
          else
            y[col] = acc[i][j][r];
        }
      }
    }
  }
}

}  // namespace

void launch_gemm_q4(const void* x, int m, int n, int k, const void* w, int epilogue, void* y,
                    hipStream_t s) {
  dim3 grid(n / BN, (m + BM - 1) / BM);
  const _Float16* X = reinterpret_cast<const _Float16*>(x);
  const uint8_t* W = reinterpret_cast<const uint8_t*>(w);
  switch (epilogue) {
    case kEpiStore:
      hipLaunchKernelGGL(gemm_q4_kernel<kEpiStore>, grid, dim3(256), 0, s, X, m, k, W, n, y);
      break;
    case kEpiAdd:
      hipLaunchKernelGGL(gemm_q4_kernel<kEpiAdd>, grid, dim3(256), 0, s, X, m, k, W, n, y);
      break;
    default:
      hipLaunchKernelGGL(gemm_q4_kernel<kEpiSwiGLU>, grid, dim3(256), 0, s, X, m, k, W, n, y);
      break;
  }
}

}  // namespace mzk
