// Causal grouped-query flash attention for gfx950 over a chunked KV cache.
//
// Queries are a sorted, possibly gappy set of absolute positions (the rows
// being recomputed); keys are every position 0..qpos of the layer, fetched
// through the layer's chunk table (chunk c lives in slot table[c]), so
// resident, restored and freshly written chunks are read in place: a single
// pass with an online softmax over non-contiguous chunks (paper Sec. 4.2),
// here on MFMA.
//
// A chunk slot stores K token-major ([C][dkv]) and V dimension-major
// ([dkv][C], "hidden-dimension-first"), so both tiles load as plain 16-byte
// rows.  A workgroup serves one KV head and a tile of query rows for all of
// that head's G query heads when G divides 8 (8 waves: G heads x 8/G groups of
// 32 rows), else for one of them (8 waves of 32 rows); each wave owns 32
// queries of one query head.  Per 64-key tile K and V^T are staged in LDS
// once for the whole workgroup, double
// buffered: the next tile's global loads are in flight while the current one
// is multiplied.  Scores are computed transposed, S^T = K Q^T,
// with v_mfma_f32_32x32x16_f16 so that each lane holds 32 scores of a single
// query: the row max needs one cross-lane exchange (lane l and l ^ 32), and
// the exponentiated scores are already laid out as the B operand of
// O^T += V^T P^T.  Softmax in fp32 with the hardware exp2 (the
// log2(e)/sqrt(hd) scale folded into one FMA); the running max is only raised
// when a tile exceeds it by more than 8 (log2 units), so rescaling the
// accumulators is rare and skipped wave-wide when no lane needs it; P (at most
// 2^8) is rounded to f16 for the MFMA, and the row sums add those same f16
// values (v_dot2 with ones, fp32 accumulation), kept per lane half and
// combined at the end.  Chunk sizes are powers of two (shift addressing).
//
// Workgroup numbering: each XCD serves one KV head (when the head count
// divides 8) and walks its query tiles heaviest (latest positions) first, so
// the 32 CUs of an XCD stream the same keys through its L2.
//
// MFMA 32x32x16 layout (checked on gfx950): lane l feeds row/column l % 32 with
// the 8 consecutive k of group l / 32; the accumulator element r of lane l is
// row 8 * (r / 4) + 4 * (l / 32) + r % 4, column l % 32.  Both operands of a
// product only need to agree on which logical k sits in (lane group, slot).
#include <algorithm>
#include <map>
#include <mutex>

#include "mz_kernels.h"

namespace mzk {
namespace {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int KT = 64;             // keys per tile
constexpr float kMaxSlack = 8.0f;  // log2 headroom before the running max is raised

// LDS tiles are unpadded and XOR-swizzled on 16-byte columns.  K tile: KT rows
// (keys) of HD halves; V^T tile: HD rows (dimensions) of KT halves (128 B).
// Row r's logical column c sits at column c ^ g(r), with g(r) = r & 15 for
// 256-byte rows and (r >> 1) & 7 for 128-byte rows: the fragment reads below
// (lane groups {0-7, 24-31}, {8-15, 16-23}, ... on 16 slots of 16 B) and the
// staging writes (8 lanes on 8 columns of one row) are bank-conflict free.
template <int ROW_HALVES>
__device__ __forceinline__ int swz(int r, int c) {
  if constexpr (ROW_HALVES == 128)
    return r * 128 + ((c ^ (r & 15)) << 3);
  else
    return r * 64 + ((c ^ ((r >> 1) & 7)) << 3);
}

// Key permutation of the score tile: MFMA row i holds key pi(i) (bits 2 and 3
// swapped), so the accumulator slots a lane turns into the P operand are 8
// consecutive keys and each V^T fragment is a single 16-byte read.
__device__ __forceinline__ int pi_key(int i) { return (i & ~0xC) | ((i & 8) >> 1) | ((i & 4) << 1); }

template <int HD>
constexpr int k_tile_halves() { return KT * HD; }
template <int HD>
constexpr int v_tile_halves() { return HD * KT; }

// SPLIT: blockIdx.y is a key split.  The workgroup covers key tiles
// [y * tps, min((y + 1) * tps, n_kt)) of its query tile and writes, per query
// row and head, the partial output normalised by its own row sum (f16, into
// Opart [split][M][nq][HD]) and (running max, row sum) (into MLpart
// [split][M][nq]; max -inf and sum 0 for a query that sees no key of the
// split).  Without SPLIT the whole key range is one pass and O is final.
// One work item: query tile `tile` (rows 32 * qw * tile ..) against KV head kvh.
template <int HD, int NW, bool DIRECT, bool SPLIT>
__device__ __forceinline__ void attn_tile(const _Float16* __restrict__ Q, const int32_t* __restrict__ qpos, int M,
                                          const uint8_t* __restrict__ slab, const int32_t* __restrict__ table,
                                          int n_table,
                                          int C, int cshift, int64_t slot_bytes, int nq, int nkv, int group,
                                          int qw, int gpw, float scale_log2, _Float16* __restrict__ O, int tps,
                                          _Float16* __restrict__ Opart, float2* __restrict__ MLpart, int tile,
                                          int kvh, int hsub0) {
  constexpr int NTH = 64 * NW;
  constexpr int KC = HD / 8;                        // 16-byte columns of a K row
  constexpr int K_SEGS = KT * KC;                   // 16-byte pieces of a K tile
  constexpr int V_SEGS = HD * (KT / 8);             // 16-byte pieces of a V^T tile
  constexpr int K_PER = (K_SEGS + NTH - 1) / NTH;
  constexpr int V_PER = (V_SEGS + NTH - 1) / NTH;
  extern __shared__ __attribute__((aligned(16))) _Float16 lds[];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int half = lane >> 5;       // lane group (0/1)
  const int col = lane & 31;        // query column of this lane
  const int dkv = nkv * HD;

  const int bq = 32 * qw;
  const int row0 = tile * bq;
  const int row_end = min(row0 + bq, M);
  const int kmax = qpos[row_end - 1];              // positions ascend
  const int kmin = qpos[row0];
  const int n_kt = kmax / KT + 1;
  // key tiles of this workgroup: [kt0, kt_end)
  const int split = SPLIT ? (int)blockIdx.y : 0;
  const int kt0 = SPLIT ? split * tps : 0;
  const int kt_end = SPLIT ? min(kt0 + tps, n_kt) : n_kt;
  if (kt0 >= kt_end) return;   // no query of this tile reaches the split

  const int h = kvh * group + hsub0 + (w % gpw);
  const bool wave_active = w < gpw * qw;
  const int qi = row0 + (w / gpw) * 32 + col;
  const bool qvalid = wave_active && qi < M;
  const int qc = min(qi, M - 1);
  const int p = qpos[qc];

  f16x8 qf[HD / 16];
  {
    const _Float16* qrow = Q + (size_t)qc * nq * HD + (wave_active ? h : 0) * HD + half * 8;
#pragma unroll
    for (int ks = 0; ks < HD / 16; ++ks) qf[ks] = *reinterpret_cast<const f16x8*>(qrow + ks * 16);
  }

  f32x16 o[HD / 32];
#pragma unroll
  for (int t = 0; t < HD / 32; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[t][r] = 0.f;
  float m_i = -INFINITY, l_i = 0.f;

  // slot layout: K [C][dkv] (token-major), then V^T [dkv][C] (dimension-major)
  const uint8_t* kbase = slab + (int64_t)kvh * HD * 2;
  const uint8_t* vbase = slab + (int64_t)C * dkv * 2 + (int64_t)kvh * HD * C * 2;
  const int cmask = C - 1;                    // C is a power of two
  const int krow_bytes = dkv * 2, vrow_bytes = C * 2;
  uint4 rk[K_PER], rv[V_PER];

  // global -> registers for K tile kt / V^T tile kt (keys past kmax are zero)
  auto gload_k = [&](int kt) {
#pragma unroll
    for (int i = 0; i < K_PER; ++i) {
      const int seg = tid + i * NTH;
      const int jj = kt * KT + seg / KC;
      rk[i] = make_uint4(0, 0, 0, 0);
      if (seg < K_SEGS && jj <= kmax)
        rk[i] = *reinterpret_cast<const uint4*>(kbase + (uint64_t)(uint32_t)table[jj >> cshift] * slot_bytes +
                                                (uint32_t)((jj & cmask) * krow_bytes + (seg % KC) * 16));
    }
  };
  auto gload_v = [&](int kt) {
#pragma unroll
    for (int i = 0; i < V_PER; ++i) {
      const int seg = tid + i * NTH;
      const int dim = seg / (KT / 8), j0 = kt * KT + (seg % (KT / 8)) * 8;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (seg < V_SEGS && j0 <= kmax) {
        // 8 keys of one chunk (C is a multiple of 8)
        v = *reinterpret_cast<const uint4*>(vbase + (uint64_t)(uint32_t)table[j0 >> cshift] * slot_bytes +
                                            (uint32_t)(dim * vrow_bytes + (j0 & cmask) * 2));
        const int nv = kmax - j0 + 1;           // keys of this group that exist
        if (nv < 8) {
          uint32_t e[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            if (2 * q >= nv) e[q] = 0u;
            else if (2 * q + 1 >= nv) e[q] &= 0xFFFFu;
          }
          v = make_uint4(e[0], e[1], e[2], e[3]);
        }
      }
      rv[i] = v;
    }
  };
  auto Kbuf = [&](int i) { return lds + (i & 1) * k_tile_halves<HD>(); };
  auto Vbuf = [&](int i) { return lds + 2 * k_tile_halves<HD>() + (i & 1) * v_tile_halves<HD>(); };
  auto lstore_k = [&](_Float16* Ks) {
#pragma unroll
    for (int i = 0; i < K_PER; ++i) {
      const int seg = tid + i * NTH;
      if (seg < K_SEGS) *reinterpret_cast<uint4*>(&Ks[swz<HD>(seg / KC, seg % KC)]) = rk[i];
    }
  };
  auto lstore_v = [&](_Float16* Vt) {
#pragma unroll
    for (int i = 0; i < V_PER; ++i) {
      const int seg = tid + i * NTH;
      if (seg < V_SEGS) *reinterpret_cast<uint4*>(&Vt[swz<KT>(seg / (KT / 8), seg % (KT / 8))]) = rv[i];
    }
  };
  // Direct path (C >= KT, so a tile lies in one chunk): the tile's slot comes
  // from one scalar table read, and each wave moves whole 1 KB stretches of
  // the swizzled LDS tile with global_load_lds_dwordx4 (lane l fills bytes
  // 16l .. 16l+15 of the stretch, so it fetches the 16 global bytes that the
  // swizzle puts there).  Per-lane offsets within a tile are loop invariant.
  constexpr int KQ = K_SEGS / 64, VQ = V_SEGS / 64;           // 1 KB stretches per tile
  constexpr int KQ_PER = (KQ + NW - 1) / NW, VQ_PER = (VQ + NW - 1) / NW;
  const int wu = __builtin_amdgcn_readfirstlane(w);
  uint32_t kofs[KQ_PER], vofs[VQ_PER];
#pragma unroll
  for (int i = 0; i < KQ_PER; ++i) {
    const int pc = (i * NW + wu) * 64 + lane;                 // 16-byte piece of the tile
    const int r = pc / KC;
    const int c = (pc % KC) ^ (HD == 128 ? (r & 15) : ((r >> 1) & 7));
    kofs[i] = (uint32_t)(r * krow_bytes + c * 16);
  }
#pragma unroll
  for (int i = 0; i < VQ_PER; ++i) {
    const int pc = (i * NW + wu) * 64 + lane;
    const int r = pc / (KT / 8);
    const int c = (pc % (KT / 8)) ^ ((r >> 1) & 7);
    vofs[i] = (uint32_t)(r * vrow_bytes + c * 16);
  }
  typedef __attribute__((address_space(3))) void lds_void;
  auto lds_addr = [&](const _Float16* p_) { return (uint32_t)(uintptr_t)(lds_void*)p_; };
  auto dload = [&](const uint8_t* gbase_, uint32_t lds0, const uint32_t* ofs, int nq_, int per) {
    // the base address is uniform: kept in scalar registers for the asm
    const uint64_t ga = (uint64_t)(uintptr_t)gbase_;
    const uint8_t* gbase = (const uint8_t*)(uintptr_t)(((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(ga >> 32)) << 32) |
                                                       (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)ga));
#pragma unroll
    for (int i = 0; i < per; ++i) {
      const int q = i * NW + wu;
      if (q < nq_)
        // one wait state between the M0 write and the load that reads it
        asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2"
                     :: "s"(lds0 + q * 1024), "v"(ofs[i]), "s"(gbase) : "memory", "m0");
    }
  };
  auto dload_k = [&](int t, const _Float16* Ks) {
    const int j0 = t * KT;
    const uint8_t* g = kbase + (uint64_t)(uint32_t)table[j0 >> cshift] * slot_bytes + (uint32_t)((j0 & cmask) * krow_bytes);
    dload(g, __builtin_amdgcn_readfirstlane(lds_addr(Ks)), kofs, KQ, KQ_PER);
  };
  auto dload_v = [&](int t, const _Float16* Vt) {
    const int j0 = t * KT;
    const uint8_t* g = vbase + (uint64_t)(uint32_t)table[j0 >> cshift] * slot_bytes + (uint32_t)((j0 & cmask) * 2);
    dload(g, __builtin_amdgcn_readfirstlane(lds_addr(Vt)), vofs, VQ, VQ_PER);
  };
  // The same with the tile's slot at hand.  Inside the key loop the slots
  // come from a copy of the item's stretch of the chunk table in LDS (ltab,
  // chunks c_lo ..): a scalar-memory read there is waited for with
  // lgkmcnt(0), two round trips per key tile before its loads can go out.
  auto dload_k_at = [&](int t, int slot, const _Float16* Ks) {
    const int j0 = t * KT;
    const uint8_t* g = kbase + (uint64_t)(uint32_t)slot * slot_bytes + (uint32_t)((j0 & cmask) * krow_bytes);
    dload(g, __builtin_amdgcn_readfirstlane(lds_addr(Ks)), kofs, KQ, KQ_PER);
  };
  auto dload_v_at = [&](int t, int slot, const _Float16* Vt) {
    const int j0 = t * KT;
    const uint8_t* g = vbase + (uint64_t)(uint32_t)slot * slot_bytes + (uint32_t)((j0 & cmask) * 2);
    dload(g, __builtin_amdgcn_readfirstlane(lds_addr(Vt)), vofs, VQ, VQ_PER);
  };
  int* ltab = reinterpret_cast<int*>(lds + 2 * (k_tile_halves<HD>() + v_tile_halves<HD>()) + 8);
  const int c_lo = (kt0 * KT) >> cshift;
  // After the wave's own loads of V^T tile t have landed: zero the keys past
  // kmax in the pieces this lane fetched (P is 0 there, but the slot rows past
  // the last written position may hold anything).
  auto vfix = [&](int t, _Float16* Vt) {
#pragma unroll
    for (int i = 0; i < VQ_PER; ++i) {
      const int q = i * NW + wu;
      if (q >= VQ) continue;
      const int pc = q * 64 + lane;
      const int r = pc / (KT / 8);
      const int c = (pc % (KT / 8)) ^ ((r >> 1) & 7);
      const int nv = kmax - (t * KT + c * 8) + 1;            // keys of this piece that exist
      if (nv < 8) {
        uint4* d = reinterpret_cast<uint4*>(Vt + pc * 8);
        uint4 v = *d;
        uint32_t e[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          if (2 * k >= nv) e[k] = 0u;
          else if (2 * k + 1 >= nv) e[k] &= 0xFFFFu;
        }
        *d = make_uint4(e[0], e[1], e[2], e[3]);
      }
    }
  };

  // S^T = K Q^T: keys (permuted by pi) on rows, this wave's 32 queries on columns
  const int krow = pi_key(col);
  auto qk = [&](const _Float16* Ks, f32x16* sc) {
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
#pragma unroll
      for (int r = 0; r < 16; ++r) sc[kk][r] = 0.f;
#pragma unroll
      for (int ks = 0; ks < HD / 16; ++ks) {
        const f16x8 a = *reinterpret_cast<const f16x8*>(&Ks[swz<HD>(kk * 32 + krow, ks * 2 + half)]);
        sc[kk] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, qf[ks], sc[kk], 0, 0, 0);
      }
    }
  };

  // causal mask of tile kt (keys past the lane's query position -> -inf).
  // Score slot (kk, r) of lane group `half` holds key
  // kt*KT + 8*half + kk*32 + 16*(r/8) + 4*((r/4)%2) + r%4 (the pi order).
  // (a bit select per score, -inf where the sign of th - c says c > th: no
  // per-score compare masks in scalar registers)
  auto mask_tile = [&](f32x16* sc, int kt) {
    const int th = p - kt * KT - 8 * half;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int c = kk * 32 + 16 * (r >> 3) + 4 * ((r >> 2) & 1) + (r & 3);
        const uint32_t m = (uint32_t)((th - c) >> 31);
        const float v = sc[kk][r];   // (a bit cast of a vector element itself reads element 0)
        sc[kk][r] = __builtin_bit_cast(float, (__builtin_bit_cast(uint32_t, v) & ~m) | (0xFF800000u & m));
      }
  };
  auto tile_max = [&](const f32x16* sc) {
    float mx = -INFINITY;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sc[kk][r]);
    return fmaxf(mx, __shfl_xor(mx, 32)) * scale_log2;
  };
  // raise the running max only when a tile exceeds it by more than the slack;
  // the accumulators are rescaled then (rare, skipped wave-wide otherwise)
  auto update_max = [&](float mx) {
    const bool raise = mx > m_i + kMaxSlack;
    const float m_new = raise ? mx : m_i;   // finite after tile 0: key 0 is visible to all
    if (__any(raise)) {
      const float alpha = exp2f(m_i - m_new);
      l_i *= alpha;
#pragma unroll
      for (int t = 0; t < HD / 32; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[t][r] *= alpha;
    }
    m_i = m_new;
  };
  // P = 2^(s * scale - m) with the raw hardware exp2 (arguments are <= 8;
  // underflow to 0 is harmless), rounded to f16 in pairs straight into the
  // MFMA B operand (pk[j] holds keys 16*j .. 16*j+15 of this lane group's
  // half, pair r of it in elements 2r, 2r+1); the row sum adds the same f16
  // values (v_dot2 with ones, fp32 accumulation).
  const f16x2 ones = {(_Float16)1.0f, (_Float16)1.0f};
  auto exp_pair = [&](const f32x16* sc, int r2, f16x8* pk) {
    const int kk = r2 >> 3, rr = r2 & 7;     // score slots 2rr, 2rr+1 of half kk
    const float e0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[kk][2 * rr], scale_log2, -m_i));
    const float e1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[kk][2 * rr + 1], scale_log2, -m_i));
    f16x8& dst = pk[r2 >> 2];
    dst[2 * (r2 & 3)] = (_Float16)e0;
    dst[2 * (r2 & 3) + 1] = (_Float16)e1;
    l_i = __builtin_amdgcn_fdot2(f16x2{dst[2 * (r2 & 3)], dst[2 * (r2 & 3) + 1]}, ones, l_i, false);
    asm volatile("" : "+v"(l_i));   // the row sum is added here, beside its exponentials
  };
  constexpr int TN = HD / 32;          // output accumulators (32 dimensions each)
  constexpr int NQK = 2 * (HD / 16);   // score MFMAs per tile (8 or 16)
  constexpr int NPV = 4 * TN;          // PV MFMAs per tile (8 or 16)
  // operand fragments: score MFMA i reads K rows of half i % 2 at k-step i / 2;
  // PV MFMA i reads V^T rows 32 * (i % TN) .. at key step i / TN
  auto kfrag = [&](const _Float16* Ks, int i) {
    return *reinterpret_cast<const f16x8*>(&Ks[swz<HD>((i & 1) * 32 + krow, (i >> 1) * 2 + half)]);
  };
  auto vfrag = [&](const _Float16* Vt, int i) {
    return *reinterpret_cast<const f16x8*>(&Vt[swz<KT>((i % TN) * 32 + col, 2 * (i / TN) + half)]);
  };
  const f32x16 zero16 = {};

  // Pipeline: K runs one tile ahead of V.  In iteration kt the LDS holds K of
  // tile kt+1 and V^T of tile kt, and the wave holds the masked scores of tile
  // kt and its running max.  Phase A issues the score MFMAs of tile kt+1, one
  // per slot, each slot also carrying a share of the exponentials of keys
  // 0-31 of tile kt; phase B issues the PV MFMAs of tile kt with the
  // exponentials of keys 32-63 and then the max of tile kt+1.  Slots are
  // fenced so the compiler keeps this order: the MFMAs of a wave then run
  // under its own VALU work.  Fragment reads run three slots ahead, each
  // issued before its slot's MFMA.  Global
  // loads of K tile kt+2 and V tile kt+1 are in flight across the iteration
  // and land in the buffers freed in iteration kt-1; one barrier per
  // iteration.
  int ts1 = 0, ts2 = 0;   // slots of key tiles kt+1 and kt+2 at the start of step kt
  if constexpr (DIRECT) {
    {
      // (a table shorter than the item's keys breaks the call's contract; the
      // copy still stays inside its LDS region)
      const int c_n = min((((kt_end - 1) * KT) >> cshift) - c_lo + 1, n_table - c_lo);
      for (int c = tid; c < c_n; c += NTH) ltab[c] = table[c_lo + c];
    }
    dload_k(kt0, Kbuf(kt0));
    dload_v(kt0, Vbuf(kt0));
    if (kt0 + 1 < kt_end) dload_k(kt0 + 1, Kbuf(kt0 + 1));
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    if (kt0 + 1 == kt_end) vfix(kt0, Vbuf(kt0));
    ts1 = table[(min(kt0 + 1, kt_end - 1) * KT) >> cshift];
    ts2 = table[(min(kt0 + 2, kt_end - 1) * KT) >> cshift];
  } else {
    gload_k(kt0);
    gload_v(kt0);
    lstore_k(Kbuf(kt0));
    lstore_v(Vbuf(kt0));
    if (kt0 + 1 < kt_end) {
      gload_k(kt0 + 1);
      lstore_k(Kbuf(kt0 + 1));
    }
  }
  __syncthreads();
  f32x16 s0[2], s1[2];
  qk(Kbuf(kt0), s0);
  if (kt0 * KT + KT - 1 > kmin) mask_tile(s0, kt0);
  update_max(tile_max(s0));
  // a query before the split's first key sees nothing here: a finite max
  // keeps its exponentials at 0 instead of NaN (its row sum stays 0)
  if constexpr (SPLIT) {
    if (m_i == -INFINITY) m_i = 0.f;
  }
  // every wave has read key tile kt0 before the first step's loads may reuse
  // its buffer
  __syncthreads();

  auto step = [&](int kt, f32x16* sc, f32x16* sn) {
    int tnext = 0;   // slot of key tile kt+3, read from ltab now, used a step later
    if constexpr (DIRECT) {
      if (kt + 2 < kt_end) dload_k_at(kt + 2, ts2, Kbuf(kt));
      if (kt + 1 < kt_end) dload_v_at(kt + 1, ts1, Vbuf(kt + 1));
      tnext = ltab[((min(kt + 3, kt_end - 1) * KT) >> cshift) - c_lo];
    } else {
      if (kt + 2 < kt_end) gload_k(kt + 2);
      if (kt + 1 < kt_end) gload_v(kt + 1);
    }
    f16x8 pk[4];
    // phase A (the score MFMAs of the last iteration read a stale buffer and
    // are discarded)
    {
      const _Float16* Kn = Kbuf(kt + 1);
      f16x8 fa = kfrag(Kn, 0), fb = kfrag(Kn, 1), fc = kfrag(Kn, 2);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < NQK; ++i) {
        const f16x8 fd = i + 3 < NQK ? kfrag(Kn, i + 3) : fc;
        __builtin_amdgcn_sched_barrier(0);   // the read goes out ahead of the MFMA
        sn[i & 1] = __builtin_amdgcn_mfma_f32_32x32x16_f16(fa, qf[i >> 1], i < 2 ? zero16 : sn[i & 1], 0, 0, 0);
        fa = fb;
        fb = fc;
        fc = fd;
        // 8 exponential pairs over the slots
        if (i % (NQK / 8) == 0) exp_pair(sc, i / (NQK / 8), pk);
        __builtin_amdgcn_sched_barrier(0);
      }
      // keep those exponentials here: they are only read in phase B
      asm volatile("" : "+v"(pk[0]), "+v"(pk[1]));
    }
    const bool more = kt + 1 < kt_end;
    if (more && (kt + 1) * KT + KT - 1 > kmin) {
      asm volatile("");   // a real branch: only the last tiles of a query block need the mask
      mask_tile(sn, kt + 1);
    }
    // phase B
    float mx = -INFINITY;
    {
      const _Float16* Vt = Vbuf(kt);
      f16x8 fa = vfrag(Vt, 0), fb = vfrag(Vt, 1), fc = vfrag(Vt, 2);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < NPV; ++i) {
        const f16x8 fd = i + 3 < NPV ? vfrag(Vt, i + 3) : fc;
        __builtin_amdgcn_sched_barrier(0);   // the read goes out ahead of the MFMA
        o[i % TN] = __builtin_amdgcn_mfma_f32_32x32x16_f16(fa, pk[i / TN], o[i % TN], 0, 0, 0);
        fa = fb;
        fb = fc;
        fc = fd;
        if (i < NPV / 2) {
          // keys 32-63 (pk[2], pk[3]) are needed from slot NPV/2 on
#pragma unroll
          for (int j = 0; j < 16 / NPV; ++j) exp_pair(sc, 8 + i * (16 / NPV) + j, pk);
        } else {
          // max of the next tile's 32 scores over the remaining slots
          constexpr int PER = 32 / (NPV / 2);
          const int b0 = (i - NPV / 2) * PER;
#pragma unroll
          for (int e = 0; e < PER; ++e) mx = fmaxf(mx, sn[(b0 + e) >> 4][(b0 + e) & 15]);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    mx = fmaxf(mx, __shfl_xor(mx, 32)) * scale_log2;
    if (more) update_max(mx);
    if constexpr (DIRECT) {
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      ts1 = ts2;
      ts2 = __builtin_amdgcn_readfirstlane(tnext);
      if (kt + 2 == kt_end) vfix(kt + 1, Vbuf(kt + 1));
    } else {
      if (kt + 2 < kt_end) lstore_k(Kbuf(kt));
      if (more) lstore_v(Vbuf(kt + 1));
    }
    __syncthreads();
  };
  int kt = kt0;
  for (; kt + 1 < kt_end; kt += 2) {
    step(kt, s0, s1);
    step(kt + 1, s1, s0);
  }
  if (kt < kt_end) step(kt, s0, s1);

  const float l = l_i + __shfl_xor(l_i, 32);
  const float inv = SPLIT ? (l > 0.f ? 1.0f / l : 0.f) : 1.0f / l;
  if constexpr (SPLIT) {
    if (qvalid && half == 0) MLpart[(size_t)(split * M + qi) * nq + h] = make_float2(l > 0.f ? m_i : -INFINITY, l);
  }
  if (qvalid) {
    _Float16* orow = SPLIT ? Opart + ((size_t)(split * M + qi) * nq + h) * HD : O + (size_t)qi * nq * HD + h * HD;
#pragma unroll
    for (int t = 0; t < HD / 32; ++t)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int dim = t * 32 + 8 * g4 + 4 * half;
        f16x4 v = {(_Float16)(o[t][4 * g4 + 0] * inv), (_Float16)(o[t][4 * g4 + 1] * inv),
                   (_Float16)(o[t][4 * g4 + 2] * inv), (_Float16)(o[t][4 * g4 + 3] * inv)};
        *reinterpret_cast<f16x4*>(orow + dim) = v;
      }
  }
}

// Work queues of the persistent form: wq[k] (k < nkv) counts the query tiles
// of KV head k handed out so far, heaviest first; wq[kWqDone] counts the
// workgroups that have finished.  They are zero when a launch starts and the
// last workgroup to finish zeroes them again.
constexpr int kWqDone = 15;
static_assert(kWqDone < kAttnQueueInts, "done counter inside the queue block");

// Next item of a persistent workgroup (thread 0): an item (query tile, or
// query tile and head) of its home KV head while that queue lasts, then the
// lightest items left in the other queues (home + 1, home + 2, ...); -1 when
// every queue is exhausted.
__device__ __forceinline__ int attn_pop(int* wq, int home, int nkv, int n_items) {
  for (int k = 0; k < nkv; ++k) {
    int qk = home + k;
    if (qk >= nkv) qk -= nkv;
    if (__hip_atomic_load(&wq[qk], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= n_items) continue;
    const int i = atomicAdd(&wq[qk], 1);
    if (i < n_items) return qk * n_items + i;
  }
  return -1;
}

// Scheduling of the work items (tile, kvh) over the workgroups (with one
// query head per workgroup an item is (tile, head of kvh's group), the heads
// of a tile in a row).
//
// Static form (wq == nullptr, and every split launch): workgroup b takes one
// item.  Workgroups are dealt to the 8 XCDs round-robin (x = b % 8).  When nkv
// divides 8, XCD x serves kv head x % nkv only, taking every (8/nkv)-th query
// tile heaviest first, so the CUs of an XCD stream the same keys and share
// them in its L2; otherwise XCD x takes tiles x, x+8, ... with all kv heads of
// a tile in a row.
//
// Persistent form (wq != nullptr, nkv divides 8, chunks of at least 64
// tokens, no key split; one workgroup per resident slot): each workgroup pops items from the queue of its XCD's KV head
// (hardware XCC id % nkv), heaviest first, so the same L2 sharing holds; an
// XCD whose queue runs dry takes the lightest tiles left in the others.  The
// XCDs run at different clocks under the power limit, and with a fixed share
// each the slowest one sets the end of the launch.
template <int HD, int NW, bool DIRECT, bool SPLIT>
__global__ __launch_bounds__(64 * NW) void attn_kernel(const _Float16* __restrict__ Q,
                                                       const int32_t* __restrict__ qpos, int M,
                                                       const uint8_t* __restrict__ slab,
                                                       const int32_t* __restrict__ table, int n_table, int C,
                                                       int cshift, int64_t slot_bytes, int nq, int nkv,
                                                       int group, int qw, int gpw, int n_items,
                                                       float scale_log2, _Float16* __restrict__ O, int tps,
                                                       _Float16* __restrict__ Opart,
                                                       float2* __restrict__ MLpart, int* __restrict__ wq) {
  // only the direct-load, unsplit instances have the persistent form
  constexpr bool kCanPersist = DIRECT && !SPLIT;
  if constexpr (!kCanPersist) {
    const int b = blockIdx.x;
    const int xcd = b % 8, j = b / 8;
    int kvh, tile_rank;
    if (8 % nkv == 0) {
      kvh = xcd % nkv;
      tile_rank = j * (8 / nkv) + xcd / nkv;
    } else {
      kvh = j % nkv;
      tile_rank = (j / nkv) * 8 + xcd;
    }
    if (tile_rank >= n_items) return;
    const int hpi = group / gpw, n_qtiles = n_items / hpi;
    attn_tile<HD, NW, DIRECT, SPLIT>(Q, qpos, M, slab, table, n_table, C, cshift, slot_bytes, nq, nkv, group, qw,
                                     gpw, scale_log2, O, tps, Opart, MLpart, n_qtiles - 1 - tile_rank / hpi, kvh,
                                     (tile_rank % hpi) * gpw);
    return;
  }
  const bool persistent = wq != nullptr;
  // the item is broadcast through the int past the K/V tiles (a static LDS
  // variable would move the tiles off their aligned base)
  extern __shared__ __attribute__((aligned(16))) _Float16 lds[];
  int& s_item = *reinterpret_cast<int*>(lds + 2 * (k_tile_halves<HD>() + v_tile_halves<HD>()));
  int home = 0;
  if (persistent) {
    unsigned xcc;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));
    home = (int)(xcc & 7) % nkv;
  }
  for (int round = 0;; ++round) {
    int kvh, tile_rank;
    if (persistent) {
      if (threadIdx.x == 0) s_item = attn_pop(wq, home, nkv, n_items);
      __syncthreads();
      const int item = __builtin_amdgcn_readfirstlane(s_item);   // uniform: item addressing stays scalar
      __syncthreads();   // every thread has the item before thread 0 pops again
      if (item < 0) break;
      kvh = item / n_items;
      tile_rank = item - kvh * n_items;
    } else {
      if (round > 0) break;
      const int b = blockIdx.x;
      const int xcd = b % 8, j = b / 8;
      if (8 % nkv == 0) {
        kvh = xcd % nkv;
        tile_rank = j * (8 / nkv) + xcd / nkv;
      } else {
        kvh = j % nkv;
        tile_rank = (j / nkv) * 8 + xcd;
      }
      if (tile_rank >= n_items) break;
    }
    const int hpi = group / gpw, n_qtiles = n_items / hpi;
    attn_tile<HD, NW, DIRECT, SPLIT>(Q, qpos, M, slab, table, n_table, C, cshift, slot_bytes, nq, nkv, group, qw,
                                     gpw, scale_log2, O, tps, Opart, MLpart, n_qtiles - 1 - tile_rank / hpi, kvh,
                                     (tile_rank % hpi) * gpw);
  }
  if (persistent && threadIdx.x == 0) {
    // no pop of this launch follows: the last workgroup zeroes the queues
    if (atomicAdd(&wq[kWqDone], 1) == (int)gridDim.x - 1) {
      for (int k = 0; k < nkv; ++k) atomicExch(&wq[k], 0);
      atomicExch(&wq[kWqDone], 0);
    }
  }
}

// Split-key attention of few query columns (decode steps and short prompts):
// a column is one (query row, query head) pair of a KV head's group, at most
// 16 of them (m rows x G heads), so the score and output products run on
// v_mfma_f32_16x16x32_f16 with the columns as the 16-wide side instead of
// padding each query row to 32 MFMA rows.  Workgroup (split, KV head): the
// split's key tiles (KT = 64 keys) in 32-key blocks; its 4 waves take blocks
// round-robin, each with its own online softmax, and combine through LDS into
// the split partial of the split kernel (f16 output normalised by its own
// sum, and (max, sum) in log2 units), so the same merge follows.
//
// Per 32-key block: S^T[keys][cols] = K Q^T as 2 (16-key) x HD/32 MFMAs with
// K fragments loaded straight from the slot rows; the accumulator holds keys
// 4 (l/16) + r (and 16 + 4 (l/16) + r for the second half) of column l%16,
// which is directly the B operand of O^T[dims][cols] += V^T P^T once the
// 32 keys are taken in that order (k slots 0-3: the first half's keys, 4-7:
// the second's); the V^T fragments are loaded in the same key order (two
// 8-byte reads of a dimension row).  Keys past the last query position hold
// whatever the slot holds: their scores are masked and their V values zeroed.
constexpr int kFewCols = 16, kFewWaves = 4, kFewBlock = 32;

template <int HD>
__global__ __launch_bounds__(64 * kFewWaves) void attn_few_kernel(
    const _Float16* __restrict__ Q, const int32_t* __restrict__ qpos, int M, const uint8_t* __restrict__ slab,
    const int32_t* __restrict__ table, int C, int cshift, int64_t slot_bytes, int nq, int nkv, int group,
    float scale_log2, int tps, _Float16* __restrict__ Opart, float2* __restrict__ MLpart) {
  constexpr int KS = HD / 32;          // 32-wide dimension steps of a score product
  constexpr int DB = HD / 16;          // 16-dimension blocks of the output
  __shared__ float s_o[kFewWaves][DB][4][64];   // per wave: O^T fragments, lane-major
  __shared__ float s_ml[kFewWaves][2][kFewCols];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int split = blockIdx.x, kvh = blockIdx.y;
  const int col = lane & 15, lg = lane >> 4;
  const int ncol = M * group;
  const bool cvalid = col < ncol;
  const int qr = cvalid ? col / group : 0, qh = kvh * group + (cvalid ? col % group : 0);
  const int p = cvalid ? qpos[qr] : -1;             // keys 0..p are seen by this column
  const int kmax = qpos[M - 1];
  const int dkv = nkv * HD;
  const int64_t krow_bytes = (int64_t)dkv * 2;
  // Q^T fragments: column col, dimensions 32 ks + 8 lg .. +8
  typedef _Float16 f16x8v __attribute__((ext_vector_type(8)));
  typedef float f32x4v __attribute__((ext_vector_type(4)));
  f16x8v bq[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    bq[ks] = f16x8v{};
    if (cvalid) bq[ks] = *reinterpret_cast<const f16x8v*>(Q + ((size_t)qr * nq + qh) * HD + ks * 32 + lg * 8);
  }
  f32x4v o[DB];
#pragma unroll
  for (int d = 0; d < DB; ++d) o[d] = f32x4v{0.f, 0.f, 0.f, 0.f};
  float m_c = -INFINITY, l_c = 0.f;
  const int nb_all = (kmax / KT + 1) * (KT / kFewBlock);      // blocks up to kmax's tile
  const int b_begin = split * tps * (KT / kFewBlock);
  // blocks b_begin + w, + kFewWaves, ... that hold a key <= kmax
  const int b_stop = min(min(b_begin + tps * (KT / kFewBlock), nb_all), kmax / kFewBlock + 1);
  const int n_w = b_begin + w < b_stop ? (b_stop - (b_begin + w) + kFewWaves - 1) / kFewWaves : 0;
  // block k of this wave, clamped to its last one (repeated loads of a valid block stand in for the
  // blocks past the end, so no branch wraps a load)
  auto blk = [&](int k) { return b_begin + w + kFewWaves * min(k, n_w - 1); };
  // K fragments of keys jc + 16 h + col (dimensions 32 ks + 8 lg .. +8) and V^T fragments of dimension
  // rows 16 d + col (keys jc + 4 lg .. +4 and jc + 16 + 4 lg .. +4) of block bb, in slot `sl`
  auto load = [&](int bb, int32_t sl, f16x8v (&ka)[2][KS], uint2 (&va)[DB][2]) {
    const uint8_t* slot = slab + (int64_t)(uint32_t)sl * slot_bytes;
    const int jc = (bb * kFewBlock) & (C - 1);
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        ka[h][ks] = *reinterpret_cast<const f16x8v*>(slot + (int64_t)(jc + h * 16 + col) * krow_bytes +
                                                      (kvh * HD + ks * 32 + lg * 8) * 2);
    const uint8_t* vt = slot + (int64_t)C * dkv * 2 + ((int64_t)(kvh * HD + col) * C + jc + 4 * lg) * 2;
#pragma unroll
    for (int d = 0; d < DB; ++d)
#pragma unroll
      for (int h = 0; h < 2; ++h) va[d][h] = *reinterpret_cast<const uint2*>(vt + (int64_t)d * 16 * C * 2 + h * 32);
  };
  auto compute = [&](int bb, f16x8v (&ka)[2][KS], uint2 (&va)[DB][2]) {
    const int j0 = bb * kFewBlock;
    f32x4v sc[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      sc[h] = f32x4v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) sc[h] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ka[h][ks], bq[ks], sc[h], 0, 0, 0);
    }
    // scale, causal mask (key j0 + 16 h + 4 lg + r against the column's position)
    float bm = -INFINITY;
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int j = j0 + h * 16 + 4 * lg + r;
        const float v = j <= p ? sc[h][r] * scale_log2 : -INFINITY;
        sc[h][r] = v;
        bm = fmaxf(bm, v);
      }
    bm = fmaxf(bm, __shfl_xor(bm, 16));
    bm = fmaxf(bm, __shfl_xor(bm, 32));
    const float m_new = fmaxf(m_c, bm);
    const float base = m_new == -INFINITY ? 0.f : m_new;   // a column that has seen no key yet
    const float alpha = exp2f(m_c - base);
    m_c = m_new;
    l_c *= alpha;
#pragma unroll
    for (int d = 0; d < DB; ++d) o[d] *= alpha;
    f16x8v pb;
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const _Float16 e = (_Float16)exp2f(sc[h][r] - base);
        pb[h * 4 + r] = e;
        l_c += (float)e;
      }
    // values of keys past the last query position are not data: zero them
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int nvk = kmax - (j0 + h * 16 + 4 * lg) + 1;   // keys of this 4-key run that exist
      if (nvk < 4) {
#pragma unroll
        for (int d = 0; d < DB; ++d) {
          uint2 v = va[d][h];
          if (nvk <= 0) v = make_uint2(0u, 0u);
          else if (nvk == 1) v = make_uint2(v.x & 0xFFFFu, 0u);
          else if (nvk == 2) v = make_uint2(v.x, 0u);
          else v = make_uint2(v.x, v.y & 0xFFFFu);
          va[d][h] = v;
        }
      }
    }
#pragma unroll
    for (int d = 0; d < DB; ++d) {
      const uint4 a4 = make_uint4(va[d][0].x, va[d][0].y, va[d][1].x, va[d][1].y);
      o[d] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8v, a4), pb, o[d], 0, 0, 0);
    }
  };
  if (n_w > 0) {
    // the next block's chunk-table entry is fetched while this block is summed, so each block waits on
    // one memory round trip (its keys and values), not two
    f16x8v ka[2][KS];
    uint2 va[DB][2];
    int32_t t_cur = table[(blk(0) * kFewBlock) >> cshift];
    for (int k = 0; k < n_w; ++k) {
      load(blk(k), t_cur, ka, va);
      t_cur = table[(blk(k + 1) * kFewBlock) >> cshift];
      compute(blk(k), ka, va);
    }
  }
  // the column's sum over its four lane groups; then the waves combine
  l_c += __shfl_xor(l_c, 16);
  l_c += __shfl_xor(l_c, 32);
  if (lg == 0) {
    s_ml[w][0][col] = m_c;
    s_ml[w][1][col] = l_c;
  }
#pragma unroll
  for (int d = 0; d < DB; ++d)
#pragma unroll
    for (int r = 0; r < 4; ++r) s_o[w][d][r][lane] = o[d][r];
  __syncthreads();
  // thread t: column t % 16, output dimensions (t / 16) * DPT .. + DPT
  static_assert(HD % (4 * kFewWaves) == 0, "output dimensions per thread");
  const int t = threadIdx.x;
  const int c = t & 15;
  if (c >= ncol) return;
  float mx = -INFINITY;
#pragma unroll
  for (int v = 0; v < kFewWaves; ++v) mx = fmaxf(mx, s_ml[v][0][c]);
  float wsum[kFewWaves], den = 0.f;
#pragma unroll
  for (int v = 0; v < kFewWaves; ++v) {
    const float mv = s_ml[v][0][c];
    wsum[v] = (mv == -INFINITY) ? 0.f : exp2f(mv - mx);
    den += wsum[v] * s_ml[v][1][c];
  }
  const int r_ = c / group, h_ = kvh * group + c % group;
  const size_t e0 = (size_t)split * M * nq + (size_t)r_ * nq + h_;
  if (t < 16) MLpart[e0] = make_float2(den > 0.f ? mx : -INFINITY, den);
  const float inv = den > 0.f ? 1.0f / den : 0.f;
  constexpr int DPT = HD / (4 * kFewWaves);    // output dimensions per thread (64 * waves / 16 threads per column)
  const int dbase = (t >> 4) * DPT;
#pragma unroll
  for (int e = 0; e < DPT; ++e) {
    const int dim = dbase + e;                 // dimension = 16 d + 4 lg' + r of a fragment lane
    const int d = dim >> 4, lg2 = (dim >> 2) & 3, r = dim & 3;
    float acc = 0.f;
#pragma unroll
    for (int v = 0; v < kFewWaves; ++v) acc += wsum[v] * s_o[v][d][r][lg2 * 16 + c];
    Opart[e0 * HD + dim] = (_Float16)(acc * inv);
  }
}

// Merge of the key splits, one workgroup per (query row, head).  With m_s,
// l_s and the normalised partial o_s of split s, and M = max m_s over the
// splits that hold keys of the query: O = sum_s 2^(m_s - M) l_s o_s / sum_s
// 2^(m_s - M) l_s.  Split 0 always holds key 0, so the denominator is
// positive; splits past the one holding the query's own position were not
// written for it: they are loaded with the others (the workspace holds every
// split) but not used.  64 lanes of output dimensions x 4 groups
// of splits (split g + 4k in group g, at most 64 splits), the group maxima,
// denominators and sums combined through LDS.
template <int HD>
__global__ __launch_bounds__(256) void attn_merge_wide_kernel(const _Float16* __restrict__ Opart,
                                                              const float2* __restrict__ MLpart,
                                                              const int32_t* __restrict__ qpos, int M, int nq,
                                                              int n_split, int tps, _Float16* __restrict__ O) {
  constexpr int DPL = HD / 64;
  __shared__ float s_m[4], s_d[4];
  __shared__ float s_acc[4][64 * DPL];
  const int e = blockIdx.x;                       // (row, head)
  const int qi = e / nq;
  const int t = threadIdx.x, dl = t & 63, sg = t >> 6;
  const size_t stride = (size_t)M * nq;
  // every load goes out at once, from split indices clamped into the
  // workspace (a branch around each load made the compiler wait for each);
  // entries past the row's splits are masked below, never used
  const int qp = qpos[qi];
  float2 ml[16];
  _Float16 pv[16][DPL];
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    const int sp = min(sg + 4 * k, n_split - 1);
    ml[k] = MLpart[sp * stride + e];
    const _Float16* p = Opart + ((size_t)sp * stride + e) * HD + dl * DPL;
#pragma unroll
    for (int q = 0; q < DPL; ++q) pv[k][q] = p[q];
  }
  const int nv = min(n_split, (qp / KT) / tps + 1);
  float mx = -INFINITY;
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    if (!(sg + 4 * k < nv && ml[k].y > 0.f)) ml[k].x = -INFINITY;
    mx = fmaxf(mx, ml[k].x);
  }
  if (dl == 0) s_m[sg] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(s_m[0], s_m[1]), fmaxf(s_m[2], s_m[3]));
  float den = 0.f, acc[DPL] = {};
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    if (ml[k].x == -INFINITY) continue;       // past the row's splits, or a range it sees nothing of
    const float wgt = exp2f(ml[k].x - mx) * ml[k].y;
    den += wgt;
#pragma unroll
    for (int q = 0; q < DPL; ++q) acc[q] = __builtin_fmaf(wgt, (float)pv[k][q], acc[q]);
  }
  if (dl == 0) s_d[sg] = den;
#pragma unroll
  for (int q = 0; q < DPL; ++q) s_acc[sg][dl * DPL + q] = acc[q];
  __syncthreads();
  if (sg == 0) {
    const float dsum = s_d[0] + s_d[1] + s_d[2] + s_d[3];
    const float inv = 1.0f / dsum;
#pragma unroll
    for (int q = 0; q < DPL; ++q) {
      const int i = dl * DPL + q;
      const float a = s_acc[0][i] + s_acc[1][i] + s_acc[2][i] + s_acc[3][i];
      O[(size_t)e * HD + i] = (_Float16)(a * inv);
    }
  }
}

// The waves of a workgroup: gpw query heads of one KV head's group times qw
// 32-row query groups, 8 waves in all: gpw is the largest divisor of the
// group size G that divides 8 (G itself when it does), and a work item is a
// (query tile, gpw of the G heads) pair.  (G waves of one row group each, for
// G = 3, 5, 6, 7, would leave SIMDs with 1 or 2 waves.)
inline void attn_wave_map(int group, int& gpw, int& qw) {
  if (group >= 8) {
    gpw = group;
    qw = 1;
    return;
  }
  gpw = 1;
  for (int g = group; g > 1; --g)
    if (group % g == 0 && 8 % g == 0) {
      gpw = g;
      break;
    }
  qw = 8 / gpw;
}

struct SplitArgs {
  int tps = 0, n_split = 1;
  _Float16* opart = nullptr;
  float2* ml = nullptr;
};

// Workgroups of one kernel instance that the whole GPU holds at once with
// lds_bytes of dynamic LDS each (cached per instance and size).
template <int HD, int NW, bool DIRECT, bool SPLIT>
int resident_wgs(size_t lds_bytes) {
  static std::mutex mu;
  static std::map<size_t, int> cache;
  std::lock_guard<std::mutex> lock(mu);
  auto it = cache.find(lds_bytes);
  if (it != cache.end()) return it->second;
  int dev = 0, cus = 0, per = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    cus = 256;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
          &per, reinterpret_cast<const void*>(&attn_kernel<HD, NW, DIRECT, SPLIT>), 64 * NW, lds_bytes) !=
          hipSuccess || per <= 0)
    per = 1;
  cache[lds_bytes] = cus * per;
  return cus * per;
}

// Dynamic LDS of a launch: the K/V tiles, double buffered, the item of the
// persistent form and, with direct loads, the copy of the chunk table.
template <int HD, bool DIRECT>
constexpr size_t attn_lds_bytes(int n_table) {
  return 2 * (k_tile_halves<HD>() + v_tile_halves<HD>()) * sizeof(_Float16) + 16 +
         (DIRECT ? 4 * (size_t)((n_table + 3) & ~3) : 0);
}

template <int HD, int NW, bool DIRECT, bool SPLIT>
void launch_nwd(const _Float16* Q, const int32_t* qpos, int m, const uint8_t* S, const int32_t* table,
               int C, int cshift, int64_t slot_bytes, int nq, int nkv, int group, int qw, int gpw, int n_table,
               float scale_log2, _Float16* O, const SplitArgs& sa, int* wq, hipStream_t s) {
  const size_t lds_bytes = attn_lds_bytes<HD, DIRECT>(n_table);
  static const bool attr = [] {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&attn_kernel<HD, NW, DIRECT, SPLIT>),
                              hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)attn_lds_bytes<HD, DIRECT>(kAttnTableMax));
    return true;
  }();
  (void)attr;
  const int bq = 32 * qw;
  // items per KV head: query tiles times the head subsets of its group
  const int n_items = (m + bq - 1) / bq * (group / gpw);
  int blocks;
  if (DIRECT && !SPLIT && wq && 8 % nkv == 0) {
    // persistent: one workgroup per resident slot, at most one per item
    blocks = (int)std::min<int64_t>((int64_t)n_items * nkv, resident_wgs<HD, NW, DIRECT, SPLIT>(lds_bytes));
  } else {
    wq = nullptr;
    // a multiple of 8, so a split's workgroups keep the XCD mapping of blockIdx.x
    blocks = (8 % nkv == 0) ? 8 * ((n_items + 8 / nkv - 1) / (8 / nkv)) : 8 * ((n_items + 7) / 8) * nkv;
  }
  hipLaunchKernelGGL((attn_kernel<HD, NW, DIRECT, SPLIT>), dim3(blocks, SPLIT ? sa.n_split : 1), dim3(64 * NW),
                     lds_bytes, s, Q, qpos, m, S, table, n_table, C, cshift, slot_bytes, nq, nkv, group, qw, gpw,
                     n_items, scale_log2, O, sa.tps, sa.opart, sa.ml, wq);
}

template <int HD, int NW, bool SPLIT>
void launch_nw(const _Float16* Q, const int32_t* qpos, int m, const uint8_t* S, const int32_t* table,
               int C, int cshift, int64_t slot_bytes, int nq, int nkv, int group, int qw, int gpw, int n_table,
               float scale_log2, _Float16* O, const SplitArgs& sa, int* wq, hipStream_t s) {
  if (C >= KT)
    launch_nwd<HD, NW, true, SPLIT>(Q, qpos, m, S, table, C, cshift, slot_bytes, nq, nkv, group, qw, gpw, n_table,
                                    scale_log2, O, sa, wq, s);
  else
    launch_nwd<HD, NW, false, SPLIT>(Q, qpos, m, S, table, C, cshift, slot_bytes, nq, nkv, group, qw, gpw, n_table,
                                     scale_log2, O, sa, wq, s);
}

template <int HD, bool SPLIT>
void launch_hd(const _Float16* Q, const int32_t* qpos, int m, const uint8_t* S, const int32_t* table,
               int C, int cshift, int64_t slot_bytes, int nq, int nkv, int group, int qw, int gpw, int n_table,
               float scale_log2, _Float16* O, const SplitArgs& sa, int* wq, hipStream_t s) {
  switch (gpw * qw) {
    case 5: launch_nw<HD, 5, SPLIT>(Q, qpos, m, S, table, C, cshift, slot_bytes, nq, nkv, group, qw, gpw, n_table, scale_log2, O, sa, wq, s); break;
    case 6: launch_nw<HD, 6, SPLIT>(Q, qpos, m, S, table, C, cshift, slot_bytes, nq, nkv, group, qw, gpw, n_table, scale_log2, O, sa, wq, s); break;
    case 7: launch_nw<HD, 7, SPLIT>(Q, qpos, m, S, table, C, cshift, slot_bytes, nq, nkv, group, qw, gpw, n_table, scale_log2, O, sa, wq, s); break;
    default: launch_nw<HD, 8, SPLIT>(Q, qpos, m, S, table, C, cshift, slot_bytes, nq, nkv, group, qw, gpw, n_table, scale_log2, O, sa, wq, s); break;
  }
}

void launch_any(const void* q, const int32_t* qpos, int m, const void* slab, const int32_t* table, int n_table,
                int chunk_tokens, int64_t slot_bytes, int n_q, int n_kv, int head_dim, void* out,
                const SplitArgs& sa, bool split, int* wq, hipStream_t s) {
  const int group = n_q / n_kv;          // 1..8
  int gpw, qw;
  attn_wave_map(group, gpw, qw);
  const float scale_log2 = 1.4426950408889634f / __builtin_sqrtf((float)head_dim);
  const _Float16* Q = reinterpret_cast<const _Float16*>(q);
  const uint8_t* S = reinterpret_cast<const uint8_t*>(slab);
  _Float16* O = reinterpret_cast<_Float16*>(out);
  int cshift = 0;
  while ((1 << cshift) < chunk_tokens) ++cshift;   // chunk_tokens is a power of two
  if (head_dim == 128) {
    if (split) launch_hd<128, true>(Q, qpos, m, S, table, chunk_tokens, cshift, slot_bytes, n_q, n_kv, group, qw, gpw, n_table, scale_log2, O, sa, nullptr, s);
    else launch_hd<128, false>(Q, qpos, m, S, table, chunk_tokens, cshift, slot_bytes, n_q, n_kv, group, qw, gpw, n_table, scale_log2, O, sa, wq, s);
  } else {
    if (split) launch_hd<64, true>(Q, qpos, m, S, table, chunk_tokens, cshift, slot_bytes, n_q, n_kv, group, qw, gpw, n_table, scale_log2, O, sa, nullptr, s);
    else launch_hd<64, false>(Q, qpos, m, S, table, chunk_tokens, cshift, slot_bytes, n_q, n_kv, group, qw, gpw, n_table, scale_log2, O, sa, wq, s);
  }
}

}  // namespace

void launch_attention(const void* q, const int32_t* qpos, int m, const void* slab,
                      const int32_t* table, int n_table, int chunk_tokens, int64_t slot_bytes, int n_q,
                      int n_kv, int head_dim, void* out, hipStream_t s, int* work_queues) {
  launch_any(q, qpos, m, slab, table, n_table, chunk_tokens, slot_bytes, n_q, n_kv, head_dim, out, SplitArgs(), false,
             work_queues, s);
}

int64_t attention_split_ws_bytes(int m, int n_q, int head_dim, int n_split) {
  const int64_t o = (int64_t)n_split * m * n_q * head_dim * 2;
  return ((o + 255) / 256) * 256 + (int64_t)n_split * m * n_q * 8;
}

int attention_split_tiles(int max_pos, int n_split) {
  const int n_kt = max_pos / KT + 1;
  return (n_kt + n_split - 1) / n_split;
}

int attention_auto_splits(int m, int max_pos, int n_q, int n_kv, int head_dim, int64_t ws_cap) {
  const int group = n_q / n_kv;
  int gpw, qw;
  attn_wave_map(group, gpw, qw);
  const int n_qtiles = (m + 32 * qw - 1) / (32 * qw);
  // workgroups per key split: one per KV head in the few-column kernel, one
  // per item and KV head in the tiled one
  const int wgs = m * group <= kFewCols ? n_kv : n_qtiles * (group / gpw) * n_kv;
  const int n_kt = max_pos / KT + 1;
  // two workgroups per CU (their LDS fits twice) over 256 CUs -- one for
  // the few-column kernel, which streams a split's keys fastest alone (8B
  // decode step, 32900 keys: 30.5 us at 31 splits against 32.0 at 58, 36.7
  // at 47 and 36.1 at 24) -- at least 4 key tiles per split, and partials
  // that fit the workspace
  constexpr int kTarget = 512, kMinTiles = 4, kMaxSplits = 64;
  const int target = m * group <= kFewCols ? kTarget / 2 : kTarget;
  if (wgs >= kTarget / 2 || n_kt < 2 * kMinTiles) return 1;
  int ns = std::min({(target + wgs - 1) / wgs, n_kt / kMinTiles, kMaxSplits});
  while (ns > 1 && attention_split_ws_bytes(m, n_q, head_dim, ns) > ws_cap) --ns;
  if (ns <= 1) return 1;
  const int tps = (n_kt + ns - 1) / ns;
  return (n_kt + tps - 1) / tps;   // no empty trailing split
}

void launch_attention_split(const void* q, const int32_t* qpos, int m, int max_pos, const void* slab,
                            const int32_t* table, int n_table, int chunk_tokens, int64_t slot_bytes, int n_q, int n_kv,
                            int head_dim, int n_split, void* ws, void* out, hipStream_t s) {
  SplitArgs sa;
  sa.tps = attention_split_tiles(max_pos, n_split);
  const int n_kt = max_pos / KT + 1;
  sa.n_split = (n_kt + sa.tps - 1) / sa.tps;
  sa.opart = reinterpret_cast<_Float16*>(ws);
  const int64_t o = (int64_t)sa.n_split * m * n_q * head_dim * 2;
  sa.ml = reinterpret_cast<float2*>(reinterpret_cast<uint8_t*>(ws) + ((o + 255) / 256) * 256);
  const int group = n_q / n_kv;
  if (m * group <= kFewCols && chunk_tokens >= kFewBlock) {
    // few query columns: one workgroup per (split, KV head) on 16-wide products
    int cshift = 0;
    while ((1 << cshift) < chunk_tokens) ++cshift;
    const float scale_log2 = 1.4426950408889634f / __builtin_sqrtf((float)head_dim);
    const dim3 grid((unsigned)sa.n_split, (unsigned)n_kv);
    const _Float16* Q = reinterpret_cast<const _Float16*>(q);
    const uint8_t* S = reinterpret_cast<const uint8_t*>(slab);
    if (head_dim == 128)
      hipLaunchKernelGGL(attn_few_kernel<128>, grid, dim3(64 * kFewWaves), 0, s, Q, qpos, m, S, table, chunk_tokens,
                         cshift, slot_bytes, n_q, n_kv, group, scale_log2, sa.tps, sa.opart, sa.ml);
    else
      hipLaunchKernelGGL(attn_few_kernel<64>, grid, dim3(64 * kFewWaves), 0, s, Q, qpos, m, S, table, chunk_tokens,
                         cshift, slot_bytes, n_q, n_kv, group, scale_log2, sa.tps, sa.opart, sa.ml);
  } else {
    launch_any(q, qpos, m, slab, table, n_table, chunk_tokens, slot_bytes, n_q, n_kv, head_dim, out, sa, true, nullptr, s);
  }
  _Float16* O = reinterpret_cast<_Float16*>(out);
  if (head_dim == 128)
    hipLaunchKernelGGL(attn_merge_wide_kernel<128>, dim3(m * n_q), dim3(256), 0, s, sa.opart, sa.ml, qpos, m, n_q,
                       sa.n_split, sa.tps, O);
  else
    hipLaunchKernelGGL(attn_merge_wide_kernel<64>, dim3(m * n_q), dim3(256), 0, s, sa.opart, sa.ml, qpos, m, n_q,
                       sa.n_split, sa.tps, O);
}

}  // namespace mzk
