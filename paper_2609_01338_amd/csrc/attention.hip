// Causal grouped-query flash attention for gfx950 over a chunked KV cache.
//
// Queries are a sorted, possibly gappy set of absolute positions (the rows
// being recomputed); keys are every position 0..qpos of the layer, fetched
// through the layer's chunk table (chunk c lives in slot table[c]), so
// resident, restored and freshly written chunks are read in place: a single
// pass with an online softmax over non-contiguous chunks (paper Sec. 4.2),
// here on MFMA.
//
// A workgroup serves one KV head and a tile of query rows for all of that
// head's G query heads; each wave owns 32 queries of one query head.  Per
// 64-key tile the keys (K rows) and the values, transposed (V^T: keys
// contiguous per dimension), are staged in LDS once for the whole group.
// Scores are computed transposed, S^T = K Q^T, with v_mfma_f32_32x32x16_f16 so
// that each lane holds 32 scores of a single query: the row max needs one
// cross-lane exchange (lane l and l ^ 32), and the exponentiated scores are
// already laid out as the B operand of O^T += V^T P^T.  Softmax in fp32 with
// exp2 and the log2(e)/sqrt(hd) scale folded in; P is rounded to f16 for the
// MFMA; the row sums are kept per lane half and combined at the end.
//
// MFMA 32x32x16 layout (checked on gfx950): lane l feeds row/column l % 32 with
// the 8 consecutive k of group l / 32; the accumulator element r of lane l is
// row 8 * (r / 4) + 4 * (l / 32) + r % 4, column l % 32.  Both operands of a
// product only need to agree on which logical k sits in (lane group, slot).
#include "mz_kernels.h"

namespace mzk {
namespace {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int KT = 64;             // keys per tile
constexpr int VT_STRIDE = KT + 4;  // halves per V^T row (136 B): conflict-free b64 reads

template <int HD>
__global__ __launch_bounds__(512) void attn_kernel(const _Float16* __restrict__ Q,
                                                   const int32_t* __restrict__ qpos, int M,
                                                   const uint8_t* __restrict__ slab,
                                                   const int32_t* __restrict__ table, int C,
                                                   int64_t slot_bytes, int nq, int nkv, int group,
                                                   int qw, float scale_log2,
                                                   _Float16* __restrict__ O) {
  constexpr int K_STRIDE = HD + 8;  // halves per K row
  __shared__ __attribute__((aligned(16))) _Float16 Ks[KT * K_STRIDE];
  __shared__ __attribute__((aligned(16))) _Float16 Vt[HD * VT_STRIDE];

  const int tid = threadIdx.x;
  const int nthreads = blockDim.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int half = lane >> 5;       // lane group (0/1)
  const int col = lane & 31;        // query column of this lane
  const int dkv = nkv * HD;
  const int kvh = blockIdx.y;
  const int bq = 32 * qw;
  const int tile = gridDim.x - 1 - blockIdx.x;     // heaviest tiles first
  const int row0 = tile * bq;
  const int row_end = min(row0 + bq, M);
  const int kmax = qpos[row_end - 1];              // positions ascend
  const int kmin = qpos[row0];
  const int n_kt = kmax / KT + 1;

  const int h = kvh * group + (w % group);
  const int qi = row0 + (w / group) * 32 + col;
  const bool qvalid = qi < M;
  const int qc = qvalid ? qi : M - 1;
  const int p = qpos[qc];

  f16x8 qf[HD / 16];
  {
    const _Float16* qrow = Q + (size_t)qc * nq * HD + h * HD + half * 8;
#pragma unroll
    for (int ks = 0; ks < HD / 16; ++ks) qf[ks] = *reinterpret_cast<const f16x8*>(qrow + ks * 16);
  }

  f32x16 o[HD / 32];
#pragma unroll
  for (int t = 0; t < HD / 32; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[t][r] = 0.f;
  float m_i = -INFINITY, l_i = 0.f;

  const uint8_t* vbase_off = slab + (int64_t)C * dkv * 2;   // V follows K inside a slot

  for (int kt = 0; kt < n_kt; ++kt) {
    __syncthreads();
    // K rows of this tile: 64 keys x HD halves in 16-byte segments
    for (int seg = tid; seg < KT * (HD / 8); seg += nthreads) {
      const int key = seg / (HD / 8), c8 = seg % (HD / 8);
      const int j = kt * KT + key;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (j <= kmax) {
        const int64_t slot = table[j / C];
        v = *reinterpret_cast<const uint4*>(slab + slot * slot_bytes +
                                            ((int64_t)(j % C) * dkv + kvh * HD + c8 * 8) * 2);
      }
      *reinterpret_cast<uint4*>(&Ks[key * K_STRIDE + c8 * 8]) = v;
    }
    // V rows, two keys at a time, written transposed as key pairs
    for (int seg = tid; seg < (KT / 2) * (HD / 8); seg += nthreads) {
      const int kp = seg % (KT / 2), dg = seg / (KT / 2);
      const int j0 = kt * KT + 2 * kp;
      uint4 v0 = make_uint4(0, 0, 0, 0), v1 = make_uint4(0, 0, 0, 0);
      if (j0 <= kmax) {
        const int64_t slot = table[j0 / C];
        v0 = *reinterpret_cast<const uint4*>(vbase_off + slot * slot_bytes +
                                             ((int64_t)(j0 % C) * dkv + kvh * HD + dg * 8) * 2);
      }
      if (j0 + 1 <= kmax) {
        const int64_t slot = table[(j0 + 1) / C];
        v1 = *reinterpret_cast<const uint4*>(
            vbase_off + slot * slot_bytes + ((int64_t)((j0 + 1) % C) * dkv + kvh * HD + dg * 8) * 2);
      }
      const uint32_t a[4] = {v0.x, v0.y, v0.z, v0.w};
      const uint32_t b[4] = {v1.x, v1.y, v1.z, v1.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        // dims dg*8 + 2i (low halves) and dg*8 + 2i + 1 (high halves)
        const uint32_t lo = (a[i] & 0xFFFFu) | (b[i] << 16);
        const uint32_t hi = (a[i] >> 16) | (b[i] & 0xFFFF0000u);
        *reinterpret_cast<uint32_t*>(&Vt[(dg * 8 + 2 * i) * VT_STRIDE + 2 * kp]) = lo;
        *reinterpret_cast<uint32_t*>(&Vt[(dg * 8 + 2 * i + 1) * VT_STRIDE + 2 * kp]) = hi;
      }
    }
    __syncthreads();

    // S^T = K Q^T: keys on rows, this wave's 32 queries on columns
    f32x16 s[2];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
#pragma unroll
      for (int r = 0; r < 16; ++r) s[kk][r] = 0.f;
#pragma unroll
      for (int ks = 0; ks < HD / 16; ++ks) {
        const f16x8 a =
            *reinterpret_cast<const f16x8*>(&Ks[(kk * 32 + col) * K_STRIDE + ks * 16 + half * 8]);
        s[kk] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, qf[ks], s[kk], 0, 0, 0);
      }
    }
    // scale, causal mask, tile max
    const bool need_mask = kt * KT + KT - 1 > kmin;
    float mx = -INFINITY;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float v = s[kk][r] * scale_log2;
        const int key = kt * KT + kk * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
        if (need_mask && key > p) v = -INFINITY;
        s[kk][r] = v;
        mx = fmaxf(mx, v);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_i, mx);       // finite: key 0 is visible to every query
    const float alpha = exp2f(m_i - m_new);
    float psum = 0.f;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float e = exp2f(s[kk][r] - m_new);
        s[kk][r] = e;
        psum += e;
      }
    l_i = l_i * alpha + psum;
    m_i = m_new;
#pragma unroll
    for (int t = 0; t < HD / 32; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[t][r] *= alpha;

    // O^T += V^T P^T over 4 steps of 16 keys.  Slot sl of lane group `half`
    // carries key 16*ks + 8*(sl/4) + 4*half + sl%4 in both operands.
#pragma unroll
    for (int ks = 0; ks < KT / 16; ++ks) {
      f16x8 pb;
#pragma unroll
      for (int sl = 0; sl < 8; ++sl) pb[sl] = (_Float16)s[ks >> 1][(ks & 1) * 8 + sl];
#pragma unroll
      for (int t = 0; t < HD / 32; ++t) {
        const _Float16* vrow = &Vt[(t * 32 + col) * VT_STRIDE + 16 * ks + 4 * half];
        const f16x4 lo = *reinterpret_cast<const f16x4*>(vrow);
        const f16x4 hi = *reinterpret_cast<const f16x4*>(vrow + 8);
        const f16x8 a = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        o[t] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, pb, o[t], 0, 0, 0);
      }
    }
  }

  const float l = l_i + __shfl_xor(l_i, 32);
  const float inv = 1.0f / l;
  if (qvalid) {
    _Float16* orow = O + (size_t)qi * nq * HD + h * HD;
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

}  // namespace

void launch_attention(const void* q, const int32_t* qpos, int m, const void* slab,
                      const int32_t* table, int chunk_tokens, int64_t slot_bytes, int n_q,
                      int n_kv, int head_dim, void* out, hipStream_t s) {
  const int group = n_q / n_kv;
  const int qw = group >= 8 ? 1 : 8 / group;        // 32-query row groups per workgroup
  const int waves = group * qw;
  const int bq = 32 * qw;
  dim3 grid((m + bq - 1) / bq, n_kv);
  const float scale_log2 = 1.4426950408889634f / __builtin_sqrtf((float)head_dim);
  const _Float16* Q = reinterpret_cast<const _Float16*>(q);
  const uint8_t* S = reinterpret_cast<const uint8_t*>(slab);
  _Float16* O = reinterpret_cast<_Float16*>(out);
  if (head_dim == 128)
    hipLaunchKernelGGL(attn_kernel<128>, grid, dim3(64 * waves), 0, s, Q, qpos, m, S, table,
                       chunk_tokens, slot_bytes, n_q, n_kv, group, qw, scale_log2, O);
  else
    hipLaunchKernelGGL(attn_kernel<64>, grid, dim3(64 * waves), 0, s, Q, qpos, m, S, table,
                       chunk_tokens, slot_bytes, n_q, n_kv, group, qw, scale_log2, O);
}

}  // namespace mzk
