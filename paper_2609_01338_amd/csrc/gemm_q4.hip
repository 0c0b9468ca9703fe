// Q4_0-weight GEMM for gfx950: Y = X . W^T, X f16 [m][k], W Q4_0 [n][k]; optionally
// Y[r] = X[a_rows[r]] . W^T (the rows of a layer that need this projection).
//
// A 512-thread workgroup computes a 256 x 256 tile of Y in 64-wide K steps.
// Eight waves in a 4 x 2 grid each own a 64 x 128 sub-tile as 4 x 8 tiles of
// v_mfma_f32_16x16x32_f16 with fp32 accumulation.  (f16 rather than bf16
// operands: same MFMA rate on this chip, three more mantissa bits, and the
// activations of this model stay far inside the f16 range.)
//
// Staging: the activation tile goes from global memory straight into LDS
// (global_load_lds_dwordx4, no registers), requested a full step before it is
// needed, in three LDS stages.  The weight tile arrives as Q4_0 (2 blocks of 32 per row: 16 code
// bytes + an fp16 scale) one step ahead in registers and is dequantized into
// one of two LDS stages.  The codes are pre-ordered (at load time) so that a
// code pair sits at bits (4m, 16 + 4m) of a dword: one v_and_or_b32 per pair
// builds two halves, 1024 + q for the pair at bits 0-3 (exponent with ulp 1)
// and 64 + q for the pair at bits 4-7 (exponent with ulp 1/16), one shift by 8
// serves the other two pairs, a packed subtract of 1032 or 72 gives q - 8
// exactly and a packed multiply by the scale gives d * (q - 8) rounded once to
// f16 (2^-11 relative): 13 VALU operations per 8 codes.  One barrier per step.
//
// LDS rows are 128 B with the 16-byte column c of row r stored at column
// c ^ ((r >> 1) & 7).  The MFMA fragment reads (rows l % 16, column l / 16)
// are conflict free.  A 16-byte store is written 8 lanes at a time into one
// 128-byte half of the 64 banks (even or odd rows), so each group of 8 lanes
// of the dequantized stores takes the two blocks of 4 rows of one parity:
// the swizzle puts their 8 pieces in 8 distinct columns (measured on gfx950:
// 8 LDS cycles per store instruction, against 16 for 8 lanes on 8
// consecutive rows).
//
// Each XCD walks a contiguous run of tiles, M-major: neighbouring tiles on one
// XCD share the activation rows in that XCD's L2 (see gemm_q4_kernel for the
// static and the persistent, work-queue form).
//
// MFMA 16x16x32 operand layout (checked on gfx950): lane l feeds row/column
// l % 16 with the 8 consecutive k of group l / 16; the accumulator holds rows
// 4 * (l / 16) + r (r = 0..3) of column l % 16.
#include <algorithm>
#include <type_traits>

#include "mz_kernels.h"
#include "rope.h"
#include "rownorm.h"

namespace mzk {
namespace {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) void glb_void;

constexpr int BN = kGemmTileN, BK = kGemmTileK;
constexpr int NT = 512;                      // threads
constexpr int ROW = BK;                      // halves per LDS row (128 B, swizzled)
constexpr int B_TILE = BN * ROW;             // one 32 KB weight stage (256 x 64)
constexpr int A_STAGES = 3, B_STAGES = 2;
constexpr int NIB_BYTES = BN * BK / 2;       // 8192

__device__ __forceinline__ float silu(float g) { return g / (1.0f + __expf(-g)); }

// LDS offset (halves) of logical 16-byte column c of row r
__device__ __forceinline__ int swz(int r, int c) { return r * ROW + ((c ^ ((r >> 1) & 7)) << 3); }

__device__ __forceinline__ uint32_t pair_code(uint32_t w, int shift) {
  // two 4-bit codes at bits [shift, shift+4) and [16+shift, 20+shift) -> halves 1024 + q
  return ((w >> shift) & 0x000F000Fu) | 0x64006400u;
}

// (x & mask) | magic in one instruction (the mask from a scalar register, the
// magic from a vector register: one scalar operand per VOP3 on this chip)
__device__ __forceinline__ uint32_t and_or(uint32_t x, uint32_t mask, uint32_t magic) {
  uint32_t r;
  asm("v_and_or_b32 %0, %1, %2, %3" : "=v"(r) : "v"(x), "s"(mask), "v"(magic));
  return r;
}

// The 8 codes of one pre-ordered dword (pair m at bits 4m and 16 + 4m) ->
// 4 f16x2 of d * (q - 8), pair m in component m.  The integer-to-half step
// is the published exponent-bias conversion of 4-bit integers (Kim et al.,
// arXiv:2211.10017): OR-ing a code into the mantissa of a half whose ulp is 1
// (or 1/16 for the high nibble) and subtracting the bias gives it exactly.
__device__ __forceinline__ uint4 dequant_dword(uint32_t w, f16x2 d2) {
  const uint32_t mag_lo = 0x64006400u;   // 1024: code bits 0-3 add q
  const uint32_t mag_hi = 0x54005400u;   // 64: code bits 4-7 add q (ulp 1/16)
  const f16x2 off_lo = {(_Float16)1032.0f, (_Float16)1032.0f};
  const f16x2 off_hi = {(_Float16)72.0f, (_Float16)72.0f};
  const uint32_t w8 = w >> 8;
  const f16x2 c0 = __builtin_bit_cast(f16x2, and_or(w, 0x000F000Fu, mag_lo));
  const f16x2 c1 = __builtin_bit_cast(f16x2, and_or(w, 0x00F000F0u, mag_hi));
  const f16x2 c2 = __builtin_bit_cast(f16x2, and_or(w8, 0x000F000Fu, mag_lo));
  const f16x2 c3 = __builtin_bit_cast(f16x2, and_or(w8, 0x00F000F0u, mag_hi));
  uint4 o;
  o.x = __builtin_bit_cast(uint32_t, (c0 - off_lo) * d2);
  o.y = __builtin_bit_cast(uint32_t, (c1 - off_hi) * d2);
  o.z = __builtin_bit_cast(uint32_t, (c2 - off_lo) * d2);
  o.w = __builtin_bit_cast(uint32_t, (c3 - off_hi) * d2);
  return o;
}

// One pre-ordered Q4_0 block (4 dwords; dword i holds elements 8i..8i+7) of
// row `row`, block `blk` -> 32 halves (logical columns 4 blk .. 4 blk + 3).
__device__ __forceinline__ void dequant_block_to_lds(uint4 nib, uint16_t dbits, _Float16* stage,
                                                     int row, int blk) {
  const _Float16 d = __builtin_bit_cast(_Float16, dbits);
  const f16x2 d2 = {d, d};
  const uint32_t w[4] = {nib.x, nib.y, nib.z, nib.w};
#pragma unroll
  for (int i = 0; i < 4; ++i)
    *reinterpret_cast<uint4*>(stage + swz(row, blk * 4 + i)) = dequant_dword(w[i], d2);
}

// Rotary-embedding epilogue of a wave's 64 x 128 (BM 256) or 16 x 128 (BM 64)
// accumulator block.  Pair partners c and c + hd/2 of a head sit in tiles j
// and j + JO (JO = hd / 32) of the same lane.  Row positions (and slot
// offsets) are read first, then the (cos, sin) of two 16-row groups at once,
// then the rotated values are stored: the table reads never wait behind the
// stores of earlier rows.
template <int EPI, int BM, int JO>
__device__ __forceinline__ void rope_epilogue(const f32x4 (&acc)[BM / 64][8], const GemmRope& ea, void* Y, int M,
                                              int mt, int nt, int wm, int wn, int col_in, int row_in) {
  constexpr int MI = BM / 64, IB = (MI >= 2 && EPI == kEpiRopeQ) ? 2 : 1;   // row groups per table read
  constexpr int HALF = JO * 16, HD = 2 * HALF;
  const int rot_end = EPI == kEpiRopeQ ? ea.n_valid : ea.n_valid >> 1;   // rotated columns
  const int col0 = nt * BN + wn * 128 + col_in;
  int pos[MI][4];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = mt * BM + wm * (BM / 4) + i * 16 + row_in + r;
      pos[i][r] = ea.pos[min(row, M - 1)];
    }
#pragma unroll
  for (int i0 = 0; i0 < MI; i0 += IB) {
    int64_t off[IB][4];
    float2 cv[IB][4][4];
#pragma unroll
    for (int ii = 0; ii < IB; ++ii)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = mt * BM + wm * (BM / 4) + (i0 + ii) * 16 + row_in + r;
        off[ii][r] = EPI == kEpiRopeKV ? ea.kv_off[min(row, M - 1)] : 0;
        const float2* cs = ea.rope_cs + (size_t)pos[i0 + ii][r] * HALF;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int j = (q / JO) * 2 * JO + q % JO;   // first-half tiles: 0..JO-1, 2JO..3JO-1, ...
          const int col = col0 + j * 16;
          cv[ii][r][q] = col < rot_end ? cs[col & (HD - 1)] : float2{0.f, 0.f};
        }
      }
#pragma unroll
    for (int ii = 0; ii < IB; ++ii)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = i0 + ii;
        const int row = mt * BM + wm * (BM / 4) + i * 16 + row_in + r;
        if (row >= M || off[ii][r] < 0) continue;  // past the rows, or a row that writes no KV
        _Float16* yr = EPI == kEpiRopeQ ? reinterpret_cast<_Float16*>(Y) + (size_t)row * ea.n_valid
                                        : reinterpret_cast<_Float16*>(ea.slab + off[ii][r]);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int j = (q / JO) * 2 * JO + q % JO;
          const int col = col0 + j * 16;
          if (col < rot_end) {
            const float x1 = acc[i][j][r], x2 = acc[i][j + JO][r];
            const float2 c = cv[ii][r][q];
            const float2 y = rope_rotate(x1, x2, c.x, c.y);
            yr[col] = (_Float16)y.x;
            yr[col + HALF] = (_Float16)y.y;
          }
        }
      }
    if constexpr (EPI == kEpiRopeKV) {
      // values: V^T[c][pos % C] of each row's slot.  A lane's 4 rows that
      // are 4 consecutive positions from a multiple of 4 in one slot (the
      // common case: recomputed chunks and prompts are runs of positions)
      // leave as one 8-byte store per column; any other row as 2-byte ones.
      const int i = i0;
      const int row0 = mt * BM + wm * (BM / 4) + i * 16 + row_in;
      bool vec = row0 + 3 < M && (pos[i][0] & 3) == 0 && off[0][0] >= 0;
#pragma unroll
      for (int r = 1; r < 4; ++r)
        vec = vec && pos[i][r] == pos[i][0] + r && off[0][r] == off[0][0] + (int64_t)r * ea.n_valid;
      if (vec) {
        const int pc = pos[i][0] & (ea.C - 1);
        uint8_t* vt = ea.slab + off[0][0] - (int64_t)pc * ea.n_valid + (int64_t)ea.C * ea.n_valid + pc * 2;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int col = col0 + j * 16;
          if (col >= rot_end && col < ea.n_valid) {
            typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
            *reinterpret_cast<f16x4*>(vt + (int64_t)(col - rot_end) * ea.C * 2) =
                f16x4{(_Float16)acc[i][j][0], (_Float16)acc[i][j][1], (_Float16)acc[i][j][2], (_Float16)acc[i][j][3]};
          }
        }
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          if (row0 + r >= M || off[0][r] < 0) continue;
          const int pc = pos[i][r] & (ea.C - 1);
          uint8_t* vt = ea.slab + off[0][r] - (int64_t)pc * ea.n_valid + (int64_t)ea.C * ea.n_valid + pc * 2;
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const int col = col0 + j * 16;
            if (col >= rot_end && col < ea.n_valid)
              *reinterpret_cast<_Float16*>(vt + (int64_t)(col - rot_end) * ea.C * 2) = (_Float16)acc[i][j][r];
          }
        }
      }
    }
  }
}

// BM = 256 (large m) or 64 (few row tiles: four times as many workgroups; the
// arithmetic of every output element is the same, so results do not depend
// on the choice).
//
// Split K (EPI == kEpiPartial): blockIdx.y is a split that takes K steps
// [y * k_steps, min((y + 1) * k_steps, K / 64)) and stores its fp32 sums in
// Y as [split][M][N]; gemm_splitk_reduce adds the splits in order and applies
// the real epilogue.
template <int EPI, int BM>
__device__ __forceinline__ void gemm_tile(const _Float16* __restrict__ X, const int32_t* __restrict__ a_rows,
                                          int M, int K, const uint8_t* __restrict__ Wp, int N,
                                          void* __restrict__ Y, int k_steps, const GemmRope& ea, int mt, int nt) {
  extern __shared__ __attribute__((aligned(16))) _Float16 lds[];
  constexpr int A_TILE = BM * ROW;                     // one activation stage
  constexpr int MI = BM / 64;                          // 16-row MFMA tiles per wave
  constexpr int RW = BM / 8;                           // activation rows loaded per wave
  _Float16* As = lds;                                  // [A_STAGES][A_TILE]
  _Float16* Bs = lds + A_STAGES * A_TILE;              // [B_STAGES][B_TILE]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave & 3, wn = wave >> 2;
  const int split = EPI == kEpiPartial ? (int)blockIdx.y : 0;
  const int ks0 = EPI == kEpiPartial ? split * k_steps : 0;
  const int nk = EPI == kEpiPartial ? min(k_steps, K / BK - ks0) : K / BK;

  // direct A loads: wave w fills rows RW*w .. RW*w+RW-1 with MI instructions
  // of 8 rows; lane l lands at LDS (row 8i + l/8, physical column l%8), which
  // holds logical column (l%8) ^ ((row >> 1) & 7).  Output row r reads
  // activation row a_rows[r] when a row list is given, else row r.
  const _Float16* a_src[MI];
#pragma unroll
  for (int i = 0; i < MI; ++i) {
    const int pr = wave * RW + i * 8 + (lane >> 3);
    const int lc = (lane & 7) ^ ((pr >> 1) & 7);
    const int r = min(mt * BM + pr, M - 1);
    a_src[i] = X + (size_t)(a_rows ? a_rows[r] : r) * K + (size_t)ks0 * BK + lc * 8;
  }
  // weight loads: one Q4_0 block per thread.  Lanes 8g..8g+7 take blocks 0
  // and 1 of rows 8 (g / 2) + (g % 2) + {0, 2, 4, 6} (one row parity, so their
  // stores stay in one bank half); a wave's loads cover 32 consecutive rows,
  // one contiguous kilobyte of codes.
  const uint8_t* wtile = Wp + ((size_t)nt * (K / BK) + ks0) * kGemmTileBytes;
  const int b_row = 8 * (tid >> 4) + ((tid >> 3) & 1) + 2 * ((tid & 7) >> 1), b_blk = tid & 1;
  const int b_idx = b_row * 2 + b_blk;

  f32x4 acc[MI][8];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // All vector-memory loads of the main loop are issued and waited for
  // explicitly.  Completion order between the direct-to-LDS loads and the
  // register loads is not relied on: every wait is a full vmcnt(0), placed
  // where only the loads about to be consumed are in flight.  The register
  // results pass through the wait as in/out operands so nothing reads them
  // before it.
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  u32x4 rnib;
  uint32_t rsc;
  const uint32_t a_lds0 = (uint32_t)(uintptr_t)(lds_void*)(As + wave * RW * ROW);
  auto load_a = [&](int kt) {            // MI direct global -> LDS loads per lane
    const uint32_t base = __builtin_amdgcn_readfirstlane(a_lds0 + (kt % A_STAGES) * A_TILE * 2);
#pragma unroll
    for (int i = 0; i < MI; ++i)
      // one wait state between the M0 write and the LDS-DMA load that reads it
      asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
                   :: "s"(base + i * 8 * ROW * 2), "v"(a_src[i] + kt * BK) : "memory", "m0");
  };
  auto load_b = [&](int kt) {
    const uint8_t* t_ = wtile + (size_t)kt * kGemmTileBytes;
    asm volatile("global_load_dwordx4 %0, %1, off" : "=v"(rnib) : "v"(t_ + b_idx * 16) : "memory");
    asm volatile("global_load_ushort %0, %1, off" : "=v"(rsc) : "v"(t_ + NIB_BYTES + b_idx * 2) : "memory");
  };
  auto dequant = [&](_Float16* stage) {
    dequant_block_to_lds(uint4{rnib.x, rnib.y, rnib.z, rnib.w}, (uint16_t)rsc, stage, b_row, b_blk);
  };

  // prologue: A of steps 0 and 1 requested, B of step 0 dequantized
  load_a(0);
  load_b(0);
  if (nk > 1) load_a(1);
  asm volatile("s_waitcnt vmcnt(0)" : "+v"(rnib), "+v"(rsc) :: "memory");
  dequant(Bs);
  __syncthreads();

  // step kt: B codes of kt+1 requested, MFMAs on stage kt, then wait for
  // B(kt+1) and A(kt+1) (requested at the end of step kt-1), dequantize
  // B(kt+1), request A(kt+2) into the stage freed by step kt-1, barrier.
  const int frag_row = lane & 15;
  const int frag_c = lane >> 4;
  for (int kt = 0; kt < nk; ++kt) {
    const bool more_b = kt + 1 < nk, more_a = kt + 2 < nk;
    if (more_b) load_b(kt + 1);
    const _Float16* Ab = As + (kt % A_STAGES) * A_TILE;
    const _Float16* Bb = Bs + (kt & 1) * B_TILE;
    if constexpr (EPI != kEpiRopeKV) {
      // every fragment of the step is requested before the first MFMA, so the
      // LDS latency of the second 32-wide half hides under the first half
      f16x8 a[BK / 32][MI], bq[BK / 32][8];
#pragma unroll
      for (int ks = 0; ks < BK / 32; ++ks) {
#pragma unroll
        for (int i = 0; i < MI; ++i)
          a[ks][i] = *reinterpret_cast<const f16x8*>(Ab + swz(wm * (BM / 4) + i * 16 + frag_row, ks * 4 + frag_c));
#pragma unroll
        for (int j = 0; j < 8; ++j)
          bq[ks][j] = *reinterpret_cast<const f16x8*>(Bb + swz(wn * 128 + j * 16 + frag_row, ks * 4 + frag_c));
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int ks = 0; ks < BK / 32; ++ks)
#pragma unroll
        for (int j = 0; j < 8; ++j)
#pragma unroll
          for (int i = 0; i < MI; ++i)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a[ks][i], bq[ks][j], acc[i][j], 0, 0, 0);
    } else {
      // the key/value epilogue needs the registers: one half at a time
#pragma unroll
      for (int ks = 0; ks < BK / 32; ++ks) {
        f16x8 a[MI];
#pragma unroll
        for (int i = 0; i < MI; ++i)
          a[i] = *reinterpret_cast<const f16x8*>(Ab + swz(wm * (BM / 4) + i * 16 + frag_row, ks * 4 + frag_c));
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const f16x8 bf =
              *reinterpret_cast<const f16x8*>(Bb + swz(wn * 128 + j * 16 + frag_row, ks * 4 + frag_c));
#pragma unroll
          for (int i = 0; i < MI; ++i)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a[i], bf, acc[i][j], 0, 0, 0);
        }
      }
    }
    if (more_b) {
      asm volatile("s_waitcnt vmcnt(0)" : "+v"(rnib), "+v"(rsc) :: "memory");
      dequant(Bs + ((kt + 1) & 1) * B_TILE);
    }
    if (more_a) load_a(kt + 2);
    __syncthreads();
  }

  // epilogue
  const int col_in = lane & 15;
  const int row_in = (lane >> 4) * 4;
  if constexpr (EPI == kEpiRopeQ || EPI == kEpiRopeKV) {
    if (ea.hd == 128)
      rope_epilogue<EPI, BM, 4>(acc, ea, Y, M, mt, nt, wm, wn, col_in, row_in);
    else if (ea.hd == 64)
      rope_epilogue<EPI, BM, 2>(acc, ea, Y, M, mt, nt, wm, wn, col_in, row_in);
    else
      rope_epilogue<EPI, BM, 1>(acc, ea, Y, M, mt, nt, wm, wn, col_in, row_in);
    return;
  }
  if constexpr (EPI == kEpiAdd) {
    // the residuals of a lane's 4 rows x 8 columns of one 16-row group are
    // read together (from rows clamped into range), and the next group's are
    // requested before this group is written back
    auto load_group = [&](int i, float (&yo)[4][8]) {
      const int row0 = mt * BM + wm * (BM / 4) + i * 16 + row_in;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float* y = reinterpret_cast<const float*>(Y) + (size_t)min(row0 + r, M - 1) * N;
#pragma unroll
        for (int j = 0; j < 8; ++j) yo[r][j] = y[nt * BN + wn * 128 + j * 16 + col_in];
      }
    };
    auto store_group = [&](int i, const float (&yo)[4][8]) {
      const int row0 = mt * BM + wm * (BM / 4) + i * 16 + row_in;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        if (row0 + r >= M) continue;
        float* y = reinterpret_cast<float*>(Y) + (size_t)(row0 + r) * N;
#pragma unroll
        for (int j = 0; j < 8; ++j) y[nt * BN + wn * 128 + j * 16 + col_in] = yo[r][j] + acc[i][j][r];
      }
    };
    float ya[4][8], yb[4][8];
    load_group(0, ya);
#pragma unroll
    for (int i = 0; i < MI; i += 2) {
      if (i + 1 < MI) load_group(i + 1, yb);
      store_group(i, ya);
      if (i + 1 < MI) {
        if (i + 2 < MI) load_group(i + 2, ya);
        store_group(i + 1, yb);
      }
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < MI; ++i) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = mt * BM + wm * (BM / 4) + i * 16 + row_in + r;
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
        float* y = reinterpret_cast<float*>(Y) + ((size_t)split * M + row) * N;
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

// Work queues of the persistent form: wq[x] counts the takers of range x so
// far, wq[kGemmWqDone] the workgroups that have finished; zero when a launch
// starts, zeroed again by the last workgroup to finish.
constexpr int kGemmWqDone = 15;
static_assert(kGemmWqDone < kGemmQueueInts, "done counter inside the queue block");

// Tile range x of the 8 XCD ranges of `total` tiles.
__device__ __forceinline__ int xcd_range_lo(int x, int total) { return (int)((int64_t)x * total / 8); }

// Next tile of a persistent workgroup (thread 0): from its XCD's own range
// while that lasts, then from the ranges of the others (home + 1, ...); -1
// when all are taken.  A counter may run past its range's length (a taker
// that found it empty); only values below the length hand out tiles.
__device__ __forceinline__ int gemm_pop(int* wq, int home, int total) {
  for (int k = 0; k < 8; ++k) {
    const int x = (home + k) & 7;
    const int lo = xcd_range_lo(x, total), len = xcd_range_lo(x + 1, total) - lo;
    const int i = atomicAdd(&wq[x], 1);
    if (i < len) return lo + i;
  }
  return -1;
}

// Scheduling of the output tiles over the workgroups.  Tile t is row tile
// t / (N / 256), column tile t % (N / 256) (M-major), and the tiles are cut
// into 8 contiguous ranges, one per XCD, so that the tiles an XCD runs at one
// time share activation rows in its L2.
//
// Static form (wq == nullptr, and every split-K launch): workgroup b takes one
// tile; workgroups are dealt to the XCDs round-robin, so XCD b % 8 walks its
// range in order.  Persistent form (wq != nullptr; one workgroup per resident
// slot): each workgroup takes the tiles of its XCD's range (hardware XCC id)
// from a counter, then those left in the other ranges.  Under the power limit
// the XCDs run at clocks several percent apart; with a fixed share each, the
// slowest one sets the end of the launch.  (Store, add and SwiGLU epilogues;
// the others always run static.)
template <int EPI, int BM>
__global__ __launch_bounds__(NT) void gemm_q4_kernel(const _Float16* __restrict__ X,
                                                     const int32_t* __restrict__ a_rows, int M, int K,
                                                     const uint8_t* __restrict__ Wp, int N,
                                                     void* __restrict__ Y, int k_steps, GemmRope ea,
                                                     int* __restrict__ wq) {
  const int n_tiles = N / BN;
  const int total = n_tiles * ((M + BM - 1) / BM);
  // the persistent form for the store, add and SwiGLU epilogues only: with
  // the RoPE epilogues the extra loop state spills inside the K loop
  constexpr bool kCanPersist = EPI == kEpiStore || EPI == kEpiAdd || EPI == kEpiSwiGLU;
  const bool persistent = kCanPersist && wq != nullptr;
  // the tile number of the persistent form passes through the first word of
  // activation stage 0, which no wave reads between tiles
  extern __shared__ __attribute__((aligned(16))) _Float16 lds[];
  int& s_item = *reinterpret_cast<int*>(lds);
  int home = 0;
  if (persistent) {
    unsigned xcc;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));
    home = (int)(xcc & 7);
  }
  for (int round = 0;; ++round) {
    int t;
    if (persistent) {
      __syncthreads();   // the previous tile is done with the LDS
      if (threadIdx.x == 0) s_item = gemm_pop(wq, home, total);
      __syncthreads();
      t = __builtin_amdgcn_readfirstlane(s_item);
      __syncthreads();   // read by every thread before the next loads land there
      if (t < 0) break;
    } else {
      if (round > 0) break;
      const int b = blockIdx.x;
      const int per = (int)gridDim.x / 8;
      t = b < per * 8 ? (b % 8) * per + b / 8 : b;
    }
    gemm_tile<EPI, BM>(X, a_rows, M, K, Wp, N, Y, k_steps, ea, t / n_tiles, t % n_tiles);
  }
  if (!persistent) return;
  if (threadIdx.x == 0 && atomicAdd(&wq[kGemmWqDone], 1) == (int)gridDim.x - 1) {
    for (int x = 0; x < 8; ++x) atomicExch(&wq[x], 0);
    atomicExch(&wq[kGemmWqDone], 0);
  }
}

// One activation row (m = 1: a decode step, the last layer's single row): the
// product of gemm_q4_kernel<kEpiPartial> without matrix cores.  Thread r of
// a 256-thread workgroup owns output column (tile row) r of n tile
// blockIdx.x; over K tiles [y * k_steps, ...) it reads that row's two code
// blocks (32 contiguous bytes: 256 threads read the tile's 8 KB of codes in
// one coalesced sweep) and two scales, up to 8 tiles ahead, decodes each code
// pair to f16 exactly as the GEMM does (one rounding of d * (q - 8)), and
// accumulates products with the f16 activations in fp32 (v_dot2).  The
// activations of each batch of tiles are staged in LDS (one pair per
// thread) and read as broadcasts.  Partials go to part [split][N] for
// gemm_splitk_reduce.  NORM: the row is RMSNorm's input, fp32 H [.][K]; each
// workgroup first takes its scale r through the norm kernel's own routine
// and stages (f16)(h * r), the values the norm kernel would have written.
constexpr int kGemvAhead = 8;     // K tiles whose codes are in flight per thread

template <bool NORM>
__global__ __launch_bounds__(256) void gemv_q4_kernel(const _Float16* __restrict__ X,
                                                      const float* __restrict__ H, float eps,
                                                      const int32_t* __restrict__ a_rows, int K,
                                                      const uint8_t* __restrict__ Wp, int N,
                                                      float* __restrict__ part, int k_steps) {
  __shared__ f16x2 xs[kGemvAhead * 32];   // 256 pairs: one per thread and batch
  const int nk = K / BK;
  const int split = blockIdx.y;
  const int kt0 = split * k_steps;
  const int kt_n = min(k_steps, nk - kt0);
  const int nt = blockIdx.x;
  const int r = threadIdx.x;
  const size_t row = a_rows ? a_rows[0] : 0;
  const _Float16* xrow = X + row * K + (size_t)kt0 * BK;
  const float* hrow = H + row * K;
  float rn = 0.f;
  if constexpr (NORM) {
    __shared__ float red[4];
    float4 v[kRowNormRegs];
    rn = row_inv_rms(hrow, K, eps, v, red);
    hrow += (size_t)kt0 * BK;
  }
  const uint8_t* tile0 = Wp + ((size_t)nt * nk + kt0) * kGemmTileBytes;
  const f16x2 off = {(_Float16)1032.0f, (_Float16)1032.0f};
  float acc = 0.f;
  for (int t0 = 0; t0 < kt_n; t0 += kGemvAhead) {
    uint4 nb[kGemvAhead][2];
    uint32_t sc[kGemvAhead];
#pragma unroll
    for (int j = 0; j < kGemvAhead; ++j) {
      if (t0 + j < kt_n) {
        const uint8_t* t = tile0 + (size_t)(t0 + j) * kGemmTileBytes;
        nb[j][0] = *reinterpret_cast<const uint4*>(t + r * 32);
        nb[j][1] = *reinterpret_cast<const uint4*>(t + r * 32 + 16);
        sc[j] = *reinterpret_cast<const uint32_t*>(t + NIB_BYTES + r * 4);
      }
    }
    __syncthreads();   // the previous batch is done with xs
    if (r < (kt_n - t0) * 32) {
      if constexpr (NORM) {
        const float2 hv = *reinterpret_cast<const float2*>(hrow + (size_t)t0 * BK + 2 * r);
        xs[r] = f16x2{norm_to_f16(hv.x, rn), norm_to_f16(hv.y, rn)};
      } else {
        xs[r] = *reinterpret_cast<const f16x2*>(xrow + (size_t)t0 * BK + 2 * r);
      }
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kGemvAhead; ++j) {
      if (t0 + j < kt_n) {
        const f16x2* xp = xs + j * 32;
#pragma unroll
        for (int blk = 0; blk < 2; ++blk) {
          const _Float16 d = __builtin_bit_cast(_Float16, (uint16_t)(sc[j] >> (16 * blk)));
          const f16x2 d2 = {d, d};
          const uint4 q = nb[j][blk];
          const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int mm = 0; mm < 4; ++mm) {
              const f16x2 c = __builtin_bit_cast(f16x2, pair_code(w[i], 4 * mm));
              const f16x2 wv = (c - off) * d2;
              acc = __builtin_amdgcn_fdot2(wv, xp[blk * 16 + 4 * i + mm], acc, false);
            }
        }
      }
    }
  }
  part[(size_t)split * N + (size_t)nt * BN + r] = acc;
}

// Sum of the K splits in split order, then the epilogue; 4 columns per
// thread (SwiGLU: 4 output columns, whose gate and up sums are 4 consecutive
// columns each: output column o takes gate column 32 (o / 16) + o % 16 and the
// up column 16 after it).
template <int EPI>
__global__ __launch_bounds__(256) void gemm_splitk_reduce(const float* __restrict__ part, int ns, int M, int N,
                                                          void* __restrict__ Y) {
  const int NO = EPI == kEpiSwiGLU ? N / 2 : N;       // output columns
  const int64_t i4 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i4 * 4 >= (int64_t)M * NO) return;
  const int row = (int)(i4 * 4 / NO), o = (int)(i4 * 4 % NO);
  const size_t plane = (size_t)M * N;
  if constexpr (EPI == kEpiSwiGLU) {
    const int cg = 32 * (o / 16) + o % 16;
    const float* pg = part + (size_t)row * N + cg;
    float4 g = *reinterpret_cast<const float4*>(pg), u = *reinterpret_cast<const float4*>(pg + 16);
    for (int sp = 1; sp < ns; ++sp) {
      const float4 g2 = *reinterpret_cast<const float4*>(pg + sp * plane);
      const float4 u2 = *reinterpret_cast<const float4*>(pg + sp * plane + 16);
      g.x += g2.x; g.y += g2.y; g.z += g2.z; g.w += g2.w;
      u.x += u2.x; u.y += u2.y; u.z += u2.z; u.w += u2.w;
    }
    _Float16* y = reinterpret_cast<_Float16*>(Y) + (size_t)row * NO + o;
    y[0] = (_Float16)(silu(g.x) * u.x);
    y[1] = (_Float16)(silu(g.y) * u.y);
    y[2] = (_Float16)(silu(g.z) * u.z);
    y[3] = (_Float16)(silu(g.w) * u.w);
  } else {
    const float* pp = part + (size_t)row * N + o;
    float4 a = *reinterpret_cast<const float4*>(pp);
    for (int sp = 1; sp < ns; ++sp) {
      const float4 b = *reinterpret_cast<const float4*>(pp + sp * plane);
      a.x += b.x; a.y += b.y; a.z += b.z; a.w += b.w;
    }
    float4* y = reinterpret_cast<float4*>(reinterpret_cast<float*>(Y) + (size_t)row * N + o);
    if (EPI == kEpiAdd) {
      const float4 c = *y;
      a.x += c.x; a.y += c.y; a.z += c.z; a.w += c.w;
    }
    *y = a;
  }
}

// Sum of the K splits in split order, then the rotary embedding of
// kEpiRopeQ / kEpiRopeKV (see GemmRope): one thread per (row, rotated pair
// c, c + hd/2) and, for keys and values, per (row, value column).
template <int EPI>
__global__ __launch_bounds__(256) void gemm_splitk_reduce_rope(const float* __restrict__ part, int ns, int M, int N,
                                                               GemmRope ea, void* __restrict__ Y) {
  const int half = ea.hd >> 1;
  const int rot = EPI == kEpiRopeQ ? ea.n_valid : ea.n_valid >> 1;   // rotated columns
  const int pairs = rot >> 1;
  const int per_row = pairs + (EPI == kEpiRopeKV ? ea.n_valid >> 1 : 0);
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= (int64_t)M * per_row) return;
  const int row = (int)(t / per_row), j = (int)(t % per_row);
  const int64_t off = EPI == kEpiRopeKV ? ea.kv_off[row] : 0;
  if (off < 0) return;                       // a row that writes no KV
  const int p = ea.pos[row];
  const size_t plane = (size_t)M * N;
  const float* pr = part + (size_t)row * N;
  if (j < pairs) {
    const int i = j % half, c = (j / half) * ea.hd + i;
    float x1 = pr[c], x2 = pr[c + half];
    for (int sp = 1; sp < ns; ++sp) {
      x1 += pr[sp * plane + c];
      x2 += pr[sp * plane + c + half];
    }
    const float2 cv = ea.rope_cs[(size_t)p * half + i];
    _Float16* yr = EPI == kEpiRopeQ ? reinterpret_cast<_Float16*>(Y) + (size_t)row * ea.n_valid
                                    : reinterpret_cast<_Float16*>(ea.slab + off);
    const float2 y = rope_rotate(x1, x2, cv.x, cv.y);
    yr[c] = (_Float16)y.x;
    yr[c + half] = (_Float16)y.y;
  } else {
    const int v = j - pairs;
    float a = pr[rot + v];
    for (int sp = 1; sp < ns; ++sp) a += pr[sp * plane + rot + v];
    const int pc = p & (ea.C - 1);
    uint8_t* vt = ea.slab + off - (int64_t)pc * ea.n_valid + (int64_t)ea.C * ea.n_valid + pc * 2;
    *reinterpret_cast<_Float16*>(vt + (int64_t)v * ea.C * 2) = (_Float16)a;
  }
}

// One activation row in one launch, with its epilogue (a decode step; a
// restore layer that carries a single row).  Workgroup g owns CPW output
// columns over the whole K range: no partials leave the workgroup and no
// second kernel runs.  Lane items are (column, Q4_0 block): 2 CPW lanes
// cover one 64-wide K tile of the CPW columns, and the 256 threads form
// S = 128 / CPW streams that take K tiles s, s + S, s + 2S, ...  A lane reads
// its block's 16 code bytes and 2-byte scale (the 2 CPW lanes of a K tile
// read 32 CPW contiguous code bytes: a column's two blocks are 32 contiguous
// bytes of the tile) and adds the block's exact code-activation products,
// then d times the block's sum, in fp32 (gemv1_dot), K tiles in increasing
// order.  The activation row is staged once in LDS with the sum of each of
// its 32-element blocks.  The 2 S partial sums of a column are then added
// in a fixed order (stream by stream, block 0 then block 1), so results are
// deterministic; they equal the split-K form's up to the order of the fp32
// sums.  NORM: the row is RMSNorm's input, fp32 H [.][K]; the workgroup first
// takes its scale through the norm kernel's own routine and stages
// (f16)(h * r), the values the norm kernel would have written.
//
// Column maps: kEpiSwiGLU takes CPW = 32 consecutive columns, the 16 gate and
// the 16 up columns of output columns 16 g .. 16 g + 15.  The rotary
// epilogues take, for workgroups of rotated columns, P = CPW / 2 pairs
// (i, i + hd / 2) of one head, so each pair is rotated where it is summed;
// the value columns of kEpiRopeKV follow as consecutive runs.
template <int EPI, int CPW>
__device__ __forceinline__ int gemv1_col(int g, int j, const GemmRope& ea) {
  if constexpr (EPI == kEpiRopeQ || EPI == kEpiRopeKV) {
    constexpr int P = CPW / 2;
    const int half = ea.hd >> 1;
    const int rot = EPI == kEpiRopeQ ? ea.n_valid : ea.n_valid >> 1;
    const int g_rot = rot / CPW;
    if (g < g_rot) {
      const int per_head = half / P;
      const int i = (g % per_head) * P + (j % P);
      return (g / per_head) * ea.hd + i + (j >= P ? half : 0);
    }
    return rot + (g - g_rot) * CPW + j;
  } else {
    return g * CPW + j;
  }
}

constexpr int kGemv1Batch = 8;    // K tiles whose codes are in flight per lane

// Codes and scales of K tiles sid + S (i0 + u), u < kGemv1Batch, of one
// lane.  Every load is issued, without a branch around it (a guarded load
// made the compiler wait for each one): positions past the stream's last
// tile reload that tile (a stream with none reloads a tile in range), and
// gemv1_dot skips them.
template <int S>
__device__ __forceinline__ void gemv1_load(const uint8_t* codes, const uint8_t* scales, int sid, int i0, int n_i,
                                           int nk, uint4 (&c)[kGemv1Batch], uint32_t (&sc)[kGemv1Batch]) {
#pragma unroll
  for (int u = 0; u < kGemv1Batch; ++u) {
    const int kt = min(max(sid + S * min(i0 + u, n_i - 1), 0), nk - 1);
    const size_t off = (size_t)kt * kGemmTileBytes;
    c[u] = *reinterpret_cast<const uint4*>(codes + off);
    sc[u] = *reinterpret_cast<const uint16_t*>(scales + off);
  }
}

// acc += the products of one lane's batch with the staged activations.  A
// block's codes are not decoded to weights: one v_and_or_b32 per code pair
// makes the pair an exact f16 integer, 1024 + q for a pair at bits 0-3 and
// 64 + q for a pair at bits 4-7 (the exponent-bias conversion of the GEMM's
// dequant without its subtract and multiply), and v_dot2 adds their exact
// products with the activations into s.  With X_lo and X_hi the sums of the
// block's activations at the two kinds of pair,
// sum_k (q_k - 8) x_k = s - (1032 X_lo + 72 X_hi), and the block's term is
// d times that, in fp32 (xc holds 1032 X_lo + 72 X_hi of every block, formed
// once per row).  9 vector operations per 8 codes instead of 17, and no
// rounding of d (q - 8) to f16.
template <int S>
__device__ __forceinline__ float gemv1_dot(const _Float16* xb, const float* xc, int blk, int sid, int i0, int n_i,
                                           const uint4 (&c)[kGemv1Batch], const uint32_t (&sc)[kGemv1Batch],
                                           float acc) {
  const uint32_t mag_lo = 0x64006400u, mag_hi = 0x54005400u;
#pragma unroll
  for (int u = 0; u < kGemv1Batch; ++u) {
    if (i0 + u < n_i) {
      const int kt = sid + S * (i0 + u);
      const float d = (float)__builtin_bit_cast(_Float16, (uint16_t)sc[u]);
      const f16x2* xp = reinterpret_cast<const f16x2*>(xb + kt * BK);
      const uint32_t w[4] = {c[u].x, c[u].y, c[u].z, c[u].w};
      float sum = 0.f;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t w8 = w[q] >> 8;
        sum = __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2, and_or(w[q], 0x000F000Fu, mag_lo)), xp[4 * q + 0],
                                     sum, false);
        sum = __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2, and_or(w[q], 0x00F000F0u, mag_hi)), xp[4 * q + 1],
                                     sum, false);
        sum = __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2, and_or(w8, 0x000F000Fu, mag_lo)), xp[4 * q + 2],
                                     sum, false);
        sum = __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2, and_or(w8, 0x00F000F0u, mag_hi)), xp[4 * q + 3],
                                     sum, false);
      }
      acc = __builtin_fmaf(d, sum - xc[2 * kt + blk], acc);
    }
  }
  return acc;
}

// Dynamic LDS of a single-row product: the staged row (K halves), then the
// correction term of each 32-element block (K / 32 floats).
constexpr size_t gemv1_lds_bytes(int k) { return (size_t)k * sizeof(_Float16) + (size_t)(k / 32) * sizeof(float); }

// LDS of the single-row products: the staged row is dynamic (K halves).
struct Gemv1Lds {
  float red[256];     // the lanes' partial sums
  float sum[32];      // the columns' sums
  float norm[4];      // block sum of the RMSNorm scale
};

// Workgroup g of one single-row product (see gemv1_kernel).
template <bool NORM, int EPI, int CPW>
__device__ __forceinline__ void gemv1_body(int g, const _Float16* __restrict__ X, const float* __restrict__ H,
                                           float eps, const int32_t* __restrict__ a_rows, int K,
                                           const uint8_t* __restrict__ Wp, void* __restrict__ Y,
                                           const GemmRope& ea, _Float16* xs, Gemv1Lds& lds) {
  constexpr int LK = 2 * CPW, S = 256 / LK;
  float* s_red = lds.red;
  float* s_sum = lds.sum;
  const int t = threadIdx.x;
  const int nk = K / BK;
  const int item = t % LK, sid = t / LK;
  const int j = item >> 1, blk = item & 1;
  const int col = gemv1_col<EPI, CPW>(g, j, ea);
  const uint8_t* wc = Wp + (size_t)(col / BN) * nk * kGemmTileBytes;
  const uint8_t* codes = wc + (col % BN) * 32 + blk * 16;
  const uint8_t* scales = wc + NIB_BYTES + (col % BN) * 4 + blk * 2;
  const int n_i = sid < nk ? (nk - sid + S - 1) / S : 0;   // K tiles of this stream
  // the first batch of weights is in flight while the row is staged
  uint4 ca[kGemv1Batch], cb[kGemv1Batch];
  uint32_t sa[kGemv1Batch], sb[kGemv1Batch];
  gemv1_load<S>(codes, scales, sid, 0, n_i, nk, ca, sa);
  // the epilogue's operands are fetched now too, each thread from an index
  // in range (threads past the epilogue's ones fetch a duplicate), so no
  // dependent load waits at the end: the residual a column adds to, and the
  // row's position, slot offset and (cos, sin) of its pair
  [[maybe_unused]] float y_old = 0.f;
  [[maybe_unused]] float2 cs_e = {};
  [[maybe_unused]] int p_e = 0;
  [[maybe_unused]] int64_t off_e = 0;
  if constexpr (EPI == kEpiAdd) y_old = reinterpret_cast<const float*>(Y)[gemv1_col<EPI, CPW>(g, t % CPW, ea)];
  if constexpr (EPI == kEpiRopeQ || EPI == kEpiRopeKV) {
    const int half = ea.hd >> 1;
    p_e = ea.pos[0];
    if constexpr (EPI == kEpiRopeKV) off_e = ea.kv_off[0];
    cs_e = ea.rope_cs[(size_t)p_e * half + gemv1_col<EPI, CPW>(g, t % (CPW / 2), ea) % half];
  }
  const size_t row = a_rows ? a_rows[0] : 0;
  if constexpr (NORM) {
    float4 v[kRowNormRegs];
    const float* hrow = H + row * K;
    const float rn = row_inv_rms(hrow, K, eps, v, lds.norm);
    const int n4 = K / 4;
#pragma unroll
    for (int k = 0; k < kRowNormRegs; ++k) {
      const int i = t + k * 256;
      if (i < n4) {
        const f16x2 a = {norm_to_f16(v[k].x, rn), norm_to_f16(v[k].y, rn)};
        const f16x2 b = {norm_to_f16(v[k].z, rn), norm_to_f16(v[k].w, rn)};
        *reinterpret_cast<uint2*>(xs + 4 * i) =
            make_uint2(__builtin_bit_cast(uint32_t, a), __builtin_bit_cast(uint32_t, b));
      }
    }
    for (int i = t + kRowNormRegs * 256; i < n4; i += 256) {
      const float4 h = reinterpret_cast<const float4*>(hrow)[i];
      const f16x2 a = {norm_to_f16(h.x, rn), norm_to_f16(h.y, rn)};
      const f16x2 b = {norm_to_f16(h.z, rn), norm_to_f16(h.w, rn)};
      *reinterpret_cast<uint2*>(xs + 4 * i) =
          make_uint2(__builtin_bit_cast(uint32_t, a), __builtin_bit_cast(uint32_t, b));
    }
  } else {
    const uint4* xr = reinterpret_cast<const uint4*>(X + row * K);
    for (int i = t; i < K / 8; i += 256) reinterpret_cast<uint4*>(xs)[i] = xr[i];
  }
  __syncthreads();   // xs staged
  // 1032 X_lo + 72 X_hi of every 32-element block of the row (gemv1_dot):
  // pair j of a block (elements 2j, 2j + 1) is of the bits-0-3 kind for even
  // j, of the bits-4-7 kind for odd j
  float* xc = reinterpret_cast<float*>(xs + K);
  for (int b = t; b < K / 32; b += 256) {
    const f16x2* xp = reinterpret_cast<const f16x2*>(xs + 32 * b);
    float x_lo = 0.f, x_hi = 0.f;
#pragma unroll
    for (int i = 0; i < 16; i += 2) {
      const f16x2 a = xp[i], h = xp[i + 1];
      x_lo += (float)a.x;
      x_lo += (float)a.y;
      x_hi += (float)h.x;
      x_hi += (float)h.y;
    }
    xc[b] = __builtin_fmaf(1032.f, x_lo, 72.f * x_hi);
  }
  __syncthreads();
  const _Float16* xb = xs + blk * 32;
  float acc = 0.f;
  // two batches in flight: the next one loads while this one is summed
  for (int i0 = 0; i0 < n_i; i0 += 2 * kGemv1Batch) {
    if (i0 + kGemv1Batch < n_i) gemv1_load<S>(codes, scales, sid, i0 + kGemv1Batch, n_i, nk, cb, sb);
    acc = gemv1_dot<S>(xb, xc, blk, sid, i0, n_i, ca, sa, acc);
    if (i0 + 2 * kGemv1Batch < n_i) gemv1_load<S>(codes, scales, sid, i0 + 2 * kGemv1Batch, n_i, nk, ca, sa);
    if (i0 + kGemv1Batch < n_i) acc = gemv1_dot<S>(xb, xc, blk, sid, i0 + kGemv1Batch, n_i, cb, sb, acc);
  }
  s_red[t] = acc;
  __syncthreads();
  if (t < CPW) {
    float a = 0.f;
#pragma unroll
    for (int s = 0; s < S; ++s) {
      a += s_red[s * LK + 2 * t];
      a += s_red[s * LK + 2 * t + 1];
    }
    s_sum[t] = a;
  }
  __syncthreads();
  if constexpr (EPI == kEpiStore || EPI == kEpiAdd) {
    if (t < CPW) {
      float* y = reinterpret_cast<float*>(Y) + gemv1_col<EPI, CPW>(g, t, ea);
      *y = EPI == kEpiAdd ? s_sum[t] + y_old : s_sum[t];
    }
  } else if constexpr (EPI == kEpiSwiGLU) {
    static_assert(CPW == 32, "SwiGLU takes the 16 gate and 16 up columns of 16 outputs");
    if (t < 16) reinterpret_cast<_Float16*>(Y)[(size_t)g * 16 + t] = (_Float16)(silu(s_sum[t]) * s_sum[t + 16]);
  } else {
    constexpr int P = CPW / 2;
    const int half = ea.hd >> 1;
    const int rot = EPI == kEpiRopeQ ? ea.n_valid : ea.n_valid >> 1;
    const int64_t off = off_e;
    if (off < 0) return;                       // the row writes no KV
    const int p = p_e;
    if (g < rot / CPW) {
      if (t < P) {
        const int c = gemv1_col<EPI, CPW>(g, t, ea);
        _Float16* yr = EPI == kEpiRopeQ ? reinterpret_cast<_Float16*>(Y) : reinterpret_cast<_Float16*>(ea.slab + off);
        const float2 y = rope_rotate(s_sum[t], s_sum[t + P], cs_e.x, cs_e.y);
        yr[c] = (_Float16)y.x;
        yr[c + half] = (_Float16)y.y;
      }
    } else if (EPI == kEpiRopeKV && t < CPW) {
      const int v = gemv1_col<EPI, CPW>(g, t, ea) - rot;
      const int pc = p & (ea.C - 1);
      uint8_t* vt = ea.slab + off - (int64_t)pc * ea.n_valid + (int64_t)ea.C * ea.n_valid + pc * 2;
      *reinterpret_cast<_Float16*>(vt + (int64_t)v * ea.C * 2) = (_Float16)s_sum[t];
    }
  }
}

template <bool NORM, int EPI, int CPW>
__global__ __launch_bounds__(256) void gemv1_kernel(const _Float16* __restrict__ X,
                                                    const float* __restrict__ H, float eps,
                                                    const int32_t* __restrict__ a_rows, int K,
                                                    const uint8_t* __restrict__ Wp, void* __restrict__ Y,
                                                    GemmRope ea) {
  extern __shared__ __align__(16) _Float16 xs[];   // the K activations of the row
  __shared__ Gemv1Lds lds;
  gemv1_body<NORM, EPI, CPW>(blockIdx.x, X, H, eps, a_rows, K, Wp, Y, ea, xs, lds);
}

// The query and the key/value projections of one row in one launch (a decode
// step): workgroups [0, g_q) are the rotary query product, the rest the
// key/value product into the chunk slot, both from the same activations.
constexpr int kGemv1QkvCols = 8;
template <bool NORM>
__global__ __launch_bounds__(256) void gemv1_qkv_kernel(int g_q, const _Float16* __restrict__ X,
                                                        const float* __restrict__ H, float eps, int K,
                                                        const int32_t* __restrict__ rows_q,
                                                        const uint8_t* __restrict__ Wq, void* __restrict__ Yq,
                                                        GemmRope eq, const int32_t* __restrict__ rows_kv,
                                                        const uint8_t* __restrict__ Wkv, GemmRope ekv) {
  extern __shared__ __align__(16) _Float16 xs[];
  __shared__ Gemv1Lds lds;
  if ((int)blockIdx.x < g_q)
    gemv1_body<NORM, kEpiRopeQ, kGemv1QkvCols>(blockIdx.x, X, H, eps, rows_q, K, Wq, Yq, eq, xs, lds);
  else
    gemv1_body<NORM, kEpiRopeKV, kGemv1QkvCols>(blockIdx.x - g_q, X, H, eps, rows_kv, K, Wkv, nullptr, ekv, xs,
                                                lds);
}

template <int BM>
constexpr size_t lds_bytes() {
  return ((size_t)A_STAGES * BM * ROW + (size_t)B_STAGES * B_TILE) * sizeof(_Float16);
}

// Rounds of resident workgroups from which a launch takes its tiles from the
// work queues (measured on the 8B projections: +3.6 % at 56 rounds, none at 8).
constexpr int kQueueMinRounds = 16;

template <int EPI, int BM>
void launch_bm(const _Float16* X, const int32_t* a_rows, int m, int n, int k, const uint8_t* W, void* y,
               hipStream_t s, int n_split = 1, int k_steps = 0, const GemmRope& ea = GemmRope{},
               int* wq = nullptr) {
  static const bool lds_ok = [] {   // more than 64 KB of dynamic LDS, once per instantiation
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_q4_kernel<EPI, BM>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_bytes<BM>());
    return true;
  }();
  (void)lds_ok;
  const int tiles = (n / BN) * ((m + BM - 1) / BM);
  int blocks = tiles;
  if (!(EPI == kEpiStore || EPI == kEpiAdd || EPI == kEpiSwiGLU) || n_split != 1) wq = nullptr;
  if (wq) {
    // persistent: one workgroup per resident slot, at most one per tile
    static const int resident = [] {
      int dev = 0, cus = 0, per = 0;
      if (hipGetDevice(&dev) != hipSuccess ||
          hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
        cus = 256;
      if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
              &per, reinterpret_cast<const void*>(&gemm_q4_kernel<EPI, BM>), NT, lds_bytes<BM>()) != hipSuccess ||
          per <= 0)
        per = 1;
      return cus * per;
    }();
    // a launch of few rounds leaves the slowest XCD less than a tile behind,
    // which moving whole tiles cannot even out: one workgroup per tile there
    if (tiles < kQueueMinRounds * resident)
      wq = nullptr;
    else
      blocks = resident;
  }
  hipLaunchKernelGGL((gemm_q4_kernel<EPI, BM>), dim3(blocks, n_split), dim3(NT), lds_bytes<BM>(), s, X, a_rows,
                     m, k, W, n, y, k_steps, ea, wq);
}

int gemm_row_tile(int m, int n) { return (n / BN) * ((m + 255) / 256) < 128 ? 64 : 256; }

int device_cus() {
  static const int cus = [] {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    return n;
  }();
  return cus;
}

// Output rows [r0, r0 + m) of the product: the row-indexed pointers (row
// list or activations, output, RoPE positions and slot offsets) are shifted.
template <int EPI, int BM>
void launch_rows(const _Float16* X, const int32_t* a_rows, int r0, int m, int n, int k, const uint8_t* W, void* y,
                 hipStream_t s, const GemmRope& ea, int* wq) {
  const _Float16* x = a_rows ? X : X + (size_t)r0 * k;
  const int32_t* ar = a_rows ? a_rows + r0 : nullptr;
  GemmRope e = ea;
  if (e.pos) e.pos += r0;
  if (e.kv_off) e.kv_off += r0;
  void* yy = y;
  if (EPI == kEpiSwiGLU)
    yy = reinterpret_cast<_Float16*>(y) + (size_t)r0 * (n / 2);
  else if (EPI == kEpiRopeQ)
    yy = reinterpret_cast<_Float16*>(y) + (size_t)r0 * ea.n_valid;
  else if (EPI == kEpiStore || EPI == kEpiAdd)
    yy = reinterpret_cast<float*>(y) + (size_t)r0 * n;
  launch_bm<EPI, BM>(x, ar, m, n, k, W, yy, s, 1, 0, e, wq);
}

// Relative duration of a 64-row tile against a 256-row one (a quarter of the
// MFMA work, the same weight traffic and dequantization).
constexpr double kTile64Cost = 0.35;

// Rows [r0, r0 + m) of the product split over K (partials in ws, then the
// reduce with the epilogue): for a remainder of few rows whose tiles alone
// would leave most of the CUs idle while each runs the whole K range.
template <int EPI>
void launch_rows_split(const _Float16* X, const int32_t* a_rows, int r0, int m, int n, int k, const uint8_t* W,
                       void* y, hipStream_t s, const GemmRope& ea, void* ws, int ns, int row_tile = 0) {
  const _Float16* x = a_rows ? X : X + (size_t)r0 * k;
  const int32_t* ar = a_rows ? a_rows + r0 : nullptr;
  GemmRope e = ea;
  if (e.pos) e.pos += r0;
  if (e.kv_off) e.kv_off += r0;
  void* yy = y;
  if (EPI == kEpiSwiGLU)
    yy = reinterpret_cast<_Float16*>(y) + (size_t)r0 * (n / 2);
  else if (EPI == kEpiRopeQ)
    yy = reinterpret_cast<_Float16*>(y) + (size_t)r0 * ea.n_valid;
  else if (EPI == kEpiStore || EPI == kEpiAdd)
    yy = reinterpret_cast<float*>(y) + (size_t)r0 * n;
  if (EPI == kEpiRopeQ || EPI == kEpiRopeKV)
    launch_gemm_q4_splitk_rope(x, m, n, k, W, EPI, e, yy, ns, ws, s, ar, nullptr, 0.f, row_tile);
  else
    launch_gemm_q4_splitk(x, m, n, k, W, EPI, yy, ns, ws, s, ar, nullptr, 0.f, row_tile);
}

template <int EPI>
void launch_epi(const _Float16* X, const int32_t* a_rows, int m, int n, int k, const uint8_t* W, void* y,
                hipStream_t s, const GemmRope& ea = GemmRope{}, int* wq = nullptr, void* ws = nullptr,
                int64_t ws_bytes = 0) {
  // 256-row tiles unless they leave most of the 256 CUs idle; then 256-row
  // tiles split over K where the K range is long, else 64-row tiles
  if (gemm_row_tile(m, n) == 64) {
    const int ns = ws ? gemm_long_k_splits(m, n, k, ws_bytes) : 1;
    if (ns > 1)
      launch_rows_split<EPI>(X, a_rows, 0, m, n, k, W, y, s, ea, ws, ns, 256);
    else
      launch_bm<EPI, 64>(X, a_rows, m, n, k, W, y, s, 1, 0, ea, wq);
    return;
  }
  // A ragged last row of 256-row tiles can make a final round of workgroups
  // that occupies few CUs (16 column tiles x 129 row tiles = 8 rounds + 16
  // workgroups on 256 CUs).  Then the whole 256-row tiles run in one launch
  // and the remaining rows as 64-row tiles in a second one.
  const int nt = n / BN, cus = device_cus();
  const int full = m / 256, rem = m - full * 256;
  if (rem > 0 && full > 0) {
    auto rounds = [&](int tiles) { return (double)((tiles + cus - 1) / cus); };
    const double one = rounds(nt * (full + 1));
    const double two = rounds(nt * full) + kTile64Cost * rounds(nt * ((rem + 63) / 64));
    if (two < one) {
      launch_rows<EPI, 256>(X, a_rows, 0, full * 256, n, k, W, y, s, ea, wq);
      // the remainder split over K when a workspace is at hand and its
      // tiles alone would not fill the chip
      const int ns = ws ? gemm_auto_splits(rem, n, k, ws_bytes) : 1;
      if (ns > 1)
        launch_rows_split<EPI>(X, a_rows, full * 256, rem, n, k, W, y, s, ea, ws, ns);
      else
        launch_rows<EPI, 64>(X, a_rows, full * 256, rem, n, k, W, y, s, ea, wq);
      return;
    }
  }
  launch_bm<EPI, 256>(X, a_rows, m, n, k, W, y, s, 1, 0, ea, wq);
}

int gemm_k_steps(int k, int n_split) {
  const int nk = k / BK;
  return (nk + n_split - 1) / n_split;
}

}  // namespace

int64_t gemm_splitk_ws_bytes(int m, int n, int n_split) { return (int64_t)n_split * m * n * 4; }

int gemm_auto_splits(int m, int n, int k, int64_t ws_cap) {
  const int bm = gemm_row_tile(m, n);
  const int tiles = (n / BN) * ((m + bm - 1) / bm);
  const int nk = k / BK;
  // about two workgroups per CU, at least 4 K steps per split.  From 1024
  // rows on, tiles that cover half the CUs run whole: there the partials and
  // their reduce cost more than the idle CUs save (K/V of 2048 rows, 1024
  // outputs, K 2048: 29.3 us whole against 31.1 in 4 splits; of 4979 rows,
  // 512 outputs, K 1536: 23.1 against 33.6)
  constexpr int kTarget = 512, kMinSteps = 4, kMaxSplits = 32, kWholeRows = 1024;
  if (tiles >= kTarget / 2 || nk < 2 * kMinSteps || (m >= kWholeRows && tiles >= kTarget / 4)) return 1;
  int ns = std::min({(kTarget + tiles - 1) / tiles, nk / kMinSteps, kMaxSplits});
  while (ns > 1 && gemm_splitk_ws_bytes(m, n, ns) > ws_cap) --ns;
  if (ns <= 1) return 1;
  const int ks = gemm_k_steps(k, ns);
  return (nk + ks - 1) / ks;   // no empty trailing split
}

int gemm_long_k_splits(int m, int n, int k, int64_t ws_cap) {
  // The 64-row tiles fill the chip, but each dequantizes its weight tiles over
  // the whole K range for 64 rows.  256-row tiles split over K into one round
  // of the chip do a quarter of that dequantization per MFMA, which pays for
  // the fp32 partials and their reduce when each split keeps at least 16 K
  // steps (2048 x 2048 x 8192: 4 splits of 32 steps).
  constexpr int kMinSteps = 16;
  const int cus = device_cus();
  const int tiles = (n / BN) * ((m + 255) / 256), nk = k / BK;
  if (tiles >= cus || (n / BN) * ((m + 63) / 64) < cus) return 1;
  const int ns = (cus + tiles - 1) / tiles;
  if (ns < 2 || nk / ns < kMinSteps || gemm_splitk_ws_bytes(m, n, ns) > ws_cap) return 1;
  const int ks = gemm_k_steps(k, ns);
  return (nk + ks - 1) / ks;
}

namespace {
// The fp32 partials [split][m][n] of a split-K product; returns the number of
// splits written.
int launch_partials(const void* x, int m, int n, int k, const void* w, int n_split, void* ws, hipStream_t s,
                    const int32_t* a_rows, const float* h_norm, float eps, int row_tile) {
  const _Float16* X = reinterpret_cast<const _Float16*>(x);
  const uint8_t* W = reinterpret_cast<const uint8_t*>(w);
  const int ks = gemm_k_steps(k, n_split);
  const int ns = (k / BK + ks - 1) / ks;
  if (h_norm)
    hipLaunchKernelGGL(gemv_q4_kernel<true>, dim3(n / BN, ns), dim3(256), 0, s, X, h_norm, eps, a_rows, k, W, n,
                       reinterpret_cast<float*>(ws), ks);
  else if (m == 1)
    hipLaunchKernelGGL(gemv_q4_kernel<false>, dim3(n / BN, ns), dim3(256), 0, s, X, nullptr, 0.f, a_rows, k, W,
                       n, reinterpret_cast<float*>(ws), ks);
  else if ((row_tile ? row_tile : gemm_row_tile(m, n)) == 64)
    launch_bm<kEpiPartial, 64>(X, a_rows, m, n, k, W, ws, s, ns, ks);
  else
    launch_bm<kEpiPartial, 256>(X, a_rows, m, n, k, W, ws, s, ns, ks);
  return ns;
}
}  // namespace

namespace {
template <bool NORM, int EPI, int CPW>
void launch_gemv1_t(const _Float16* X, int n, int k, const uint8_t* W, const GemmRope& ea, void* y, hipStream_t s,
                    const int32_t* a_rows, const float* h, float eps) {
  const int cols = (EPI == kEpiRopeQ || EPI == kEpiRopeKV) ? ea.n_valid : n;
  hipLaunchKernelGGL((gemv1_kernel<NORM, EPI, CPW>), dim3(cols / CPW), dim3(256), gemv1_lds_bytes(k), s,
                     X, h, eps, a_rows, k, W, y, ea);
}

// Columns per workgroup: 32 for SwiGLU (gate and up of 16 outputs), else 16
// when that still gives at least 512 workgroups (two per CU), else 8.
template <int EPI>
void launch_gemv1_e(const _Float16* X, int n, int k, const uint8_t* W, const GemmRope& ea, void* y, hipStream_t s,
                    const int32_t* a_rows, const float* h, float eps) {
  const int cols = (EPI == kEpiRopeQ || EPI == kEpiRopeKV) ? ea.n_valid : n;
  if constexpr (EPI == kEpiSwiGLU) {
    if (h) launch_gemv1_t<true, EPI, 32>(X, n, k, W, ea, y, s, a_rows, h, eps);
    else launch_gemv1_t<false, EPI, 32>(X, n, k, W, ea, y, s, a_rows, h, eps);
  } else if (cols / 16 >= 512) {
    if (h) launch_gemv1_t<true, EPI, 16>(X, n, k, W, ea, y, s, a_rows, h, eps);
    else launch_gemv1_t<false, EPI, 16>(X, n, k, W, ea, y, s, a_rows, h, eps);
  } else {
    if (h) launch_gemv1_t<true, EPI, 8>(X, n, k, W, ea, y, s, a_rows, h, eps);
    else launch_gemv1_t<false, EPI, 8>(X, n, k, W, ea, y, s, a_rows, h, eps);
  }
}
}  // namespace

void launch_gemv1_qkv(const void* x, int k, const void* wq, void* yq, const GemmRope& eq, const int32_t* rows_q,
                      const void* wkv, const GemmRope& ekv, const int32_t* rows_kv, hipStream_t s,
                      const float* h_norm, float eps) {
  const _Float16* X = reinterpret_cast<const _Float16*>(x);
  const int g_q = eq.n_valid / kGemv1QkvCols, g_kv = ekv.n_valid / kGemv1QkvCols;
  const size_t lds = gemv1_lds_bytes(k);
  const uint8_t* Wq = reinterpret_cast<const uint8_t*>(wq);
  const uint8_t* Wkv = reinterpret_cast<const uint8_t*>(wkv);
  if (h_norm)
    hipLaunchKernelGGL(gemv1_qkv_kernel<true>, dim3(g_q + g_kv), dim3(256), lds, s, g_q, X, h_norm, eps, k, rows_q,
                       Wq, yq, eq, rows_kv, Wkv, ekv);
  else
    hipLaunchKernelGGL(gemv1_qkv_kernel<false>, dim3(g_q + g_kv), dim3(256), lds, s, g_q, X, h_norm, eps, k, rows_q,
                       Wq, yq, eq, rows_kv, Wkv, ekv);
}

bool gemv1_ok(int n, int k) { return n > 0 && k > 0 && n % BN == 0 && k % BK == 0 && k <= kGemv1MaxK; }

void launch_gemv1(const void* x, int n, int k, const void* w, int epilogue, const GemmRope& ea, void* y,
                  hipStream_t s, const int32_t* a_rows, const float* h_norm, float eps) {
  const _Float16* X = reinterpret_cast<const _Float16*>(x);
  const uint8_t* W = reinterpret_cast<const uint8_t*>(w);
  switch (epilogue) {
    case kEpiStore: launch_gemv1_e<kEpiStore>(X, n, k, W, ea, y, s, a_rows, h_norm, eps); break;
    case kEpiAdd: launch_gemv1_e<kEpiAdd>(X, n, k, W, ea, y, s, a_rows, h_norm, eps); break;
    case kEpiSwiGLU: launch_gemv1_e<kEpiSwiGLU>(X, n, k, W, ea, y, s, a_rows, h_norm, eps); break;
    case kEpiRopeQ: launch_gemv1_e<kEpiRopeQ>(X, n, k, W, ea, y, s, a_rows, h_norm, eps); break;
    default: launch_gemv1_e<kEpiRopeKV>(X, n, k, W, ea, y, s, a_rows, h_norm, eps); break;
  }
}

void launch_gemm_q4_splitk_rope(const void* x, int m, int n, int k, const void* w, int epilogue, const GemmRope& ea,
                                void* y, int n_split, void* ws, hipStream_t s, const int32_t* a_rows,
                                const float* h_norm, float eps, int row_tile) {
  const int ns = launch_partials(x, m, n, k, w, n_split, ws, s, a_rows, h_norm, eps, row_tile);
  const int rot = epilogue == kEpiRopeQ ? ea.n_valid : ea.n_valid / 2;
  const int64_t per_row = rot / 2 + (epilogue == kEpiRopeKV ? ea.n_valid / 2 : 0);
  const dim3 grid((unsigned)(((int64_t)m * per_row + 255) / 256));
  const float* part = reinterpret_cast<const float*>(ws);
  if (epilogue == kEpiRopeQ)
    hipLaunchKernelGGL(gemm_splitk_reduce_rope<kEpiRopeQ>, grid, dim3(256), 0, s, part, ns, m, n, ea, y);
  else
    hipLaunchKernelGGL(gemm_splitk_reduce_rope<kEpiRopeKV>, grid, dim3(256), 0, s, part, ns, m, n, ea, y);
}

void launch_gemm_q4_splitk(const void* x, int m, int n, int k, const void* w, int epilogue, void* y, int n_split,
                           void* ws, hipStream_t s, const int32_t* a_rows, const float* h_norm, float eps,
                           int row_tile) {
  const int ns = launch_partials(x, m, n, k, w, n_split, ws, s, a_rows, h_norm, eps, row_tile);
  const int64_t outs = (int64_t)m * (epilogue == kEpiSwiGLU ? n / 2 : n) / 4;
  const dim3 grid((unsigned)((outs + 255) / 256));
  const float* part = reinterpret_cast<const float*>(ws);
  switch (epilogue) {
    case kEpiStore: hipLaunchKernelGGL(gemm_splitk_reduce<kEpiStore>, grid, dim3(256), 0, s, part, ns, m, n, y); break;
    case kEpiAdd: hipLaunchKernelGGL(gemm_splitk_reduce<kEpiAdd>, grid, dim3(256), 0, s, part, ns, m, n, y); break;
    default: hipLaunchKernelGGL(gemm_splitk_reduce<kEpiSwiGLU>, grid, dim3(256), 0, s, part, ns, m, n, y); break;
  }
}

void launch_gemm_q4(const void* x, int m, int n, int k, const void* w, int epilogue, void* y,
                    hipStream_t s, const int32_t* a_rows, int* work_queues, void* ws, int64_t ws_bytes) {
  const _Float16* X = reinterpret_cast<const _Float16*>(x);
  const uint8_t* W = reinterpret_cast<const uint8_t*>(w);
  switch (epilogue) {
    case kEpiStore: launch_epi<kEpiStore>(X, a_rows, m, n, k, W, y, s, GemmRope{}, work_queues, ws, ws_bytes); break;
    case kEpiAdd: launch_epi<kEpiAdd>(X, a_rows, m, n, k, W, y, s, GemmRope{}, work_queues, ws, ws_bytes); break;
    default: launch_epi<kEpiSwiGLU>(X, a_rows, m, n, k, W, y, s, GemmRope{}, work_queues, ws, ws_bytes); break;
  }
}

bool gemm_rope_fusable(int head_dim, int chunk_tokens) {
  return (head_dim == 32 || head_dim == 64 || head_dim == 128) && chunk_tokens > 0 &&
         (chunk_tokens & (chunk_tokens - 1)) == 0;
}

void launch_gemm_q4_rope(const void* x, int m, int n, int k, const void* w, int epilogue, const GemmRope& ea,
                         void* y, hipStream_t s, const int32_t* a_rows, int* work_queues, void* ws,
                         int64_t ws_bytes) {
  const _Float16* X = reinterpret_cast<const _Float16*>(x);
  const uint8_t* W = reinterpret_cast<const uint8_t*>(w);
  if (epilogue == kEpiRopeQ)
    launch_epi<kEpiRopeQ>(X, a_rows, m, n, k, W, y, s, ea, work_queues, ws, ws_bytes);
  else
    launch_epi<kEpiRopeKV>(X, a_rows, m, n, k, W, y, s, ea, work_queues, ws, ws_bytes);
}

}  // namespace mzk
