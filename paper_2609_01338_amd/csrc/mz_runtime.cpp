// Runtime and C ABI of the restore-and-prefill engine (see include/mz.h).
//
// Memory (paper Sec. 4.2, re-targeted to a discrete GPU):
//  - KV: one HBM slab of fixed-size slots, one slot per (layer, chunk), each
//    holding K of chunk_tokens tokens token-major ([C][dkv] f16) and then V
//    dimension-major ([dkv][C] f16: the chunk is "hidden-dimension-first" for
//    the values, which the attention kernel stages without transposing).  A per-layer
//    chunk table maps chunk -> slot; free slots sit in an ordered set so that
//    contiguous runs can be handed out for coalesced copies.  Allocation at
//    restore time is O(log n) with no driver call.
//  - Weights: one unit per layer (fused QKV, O, gate/up interleaved, down, all
//    in the tiled GEMM layout) in a pool of equal-size unit slots; embedding
//    and output head are never evicted.
//  - Swap space: a stack of pinned host segments; eviction pushes units in
//    plan order (backward-out by default) and restoration reads them back
//    forward-in (Sec. 4.4).
// Restore (Sec. 4.4, 5): a host planner derives the rows R_l that must pass
// through each layer and the rows D_l whose K/V is written, allocates slots,
// uploads the row metadata, issues the swap-in copies on a side stream with
// one event per layer and kind, and enqueues the per-layer kernels on the
// compute stream, which waits on a layer's events only right before the first
// kernel that reads the restored data.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <exception>
#include <memory>
#include <set>
#include <string>
#include <thread>
#include <vector>

#include "../../include/mz.h"
#include "mz_internal.h"
#include "mz_kernels.h"

namespace {

constexpr const char* kVersion = "mz-mi355x 0.1";

thread_local std::string g_load_error;

struct HipError {
  hipError_t e;
  const char* what;
};

#define HIPCHK(x)                                      \
  do {                                                 \
    hipError_t e_ = (x);                               \
    if (e_ != hipSuccess) throw HipError{e_, #x};      \
  } while (0)

struct StatusError {
  mz_status st;
  std::string msg;
};

[[noreturn]] void fail(mz_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  throw StatusError{st, buf};
}

int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

// ---------------------------------------------------------------- weight unit layout

struct UnitLayout {
  int64_t off_q, off_kv, off_o, off_gu, off_dn, unit_bytes;
};

int64_t gemm_packed_bytes(int64_t n, int64_t k);

UnitLayout unit_layout(const mz_model_cfg& cfg) {
  const int64_t d = cfg.d_model, dq = (int64_t)cfg.n_q_heads * cfg.head_dim,
                dkv = (int64_t)cfg.n_kv_heads * cfg.head_dim,
                ffp = round_up(cfg.d_ffn, mzk::kGemmTileN / 2);
  const int64_t b_q = gemm_packed_bytes(dq, d), b_kv = gemm_packed_bytes(2 * dkv, d),
                b_o = gemm_packed_bytes(d, dq), b_gu = gemm_packed_bytes(2 * ffp, d),
                b_dn = gemm_packed_bytes(d, ffp);
  UnitLayout u;
  u.off_q = 0;
  u.off_kv = round_up(b_q, 256);
  u.off_o = u.off_kv + round_up(b_kv, 256);
  u.off_gu = u.off_o + round_up(b_o, 256);
  u.off_dn = u.off_gu + round_up(b_gu, 256);
  u.unit_bytes = round_up(u.off_dn + b_dn, 4096);
  return u;
}

// ---------------------------------------------------------------- Q4_0 repacking

constexpr int kBlockBytes = 18;

int64_t q4_row_bytes(int64_t cols) { return (cols + 31) / 32 * kBlockBytes; }

int64_t gemm_packed_bytes(int64_t n, int64_t k) {
  return round_up(n, mzk::kGemmTileN) / mzk::kGemmTileN * (round_up(k, mzk::kGemmTileK) / mzk::kGemmTileK) *
         mzk::kGemmTileBytes;
}

// Codes of one block (element j in the low nibble of byte j, element j+16 in
// its high nibble) re-ordered for the GEMM's dequantizer: dword i carries
// elements 8i..8i+7, element 8i+2m at bits 4m and element 8i+2m+1 at bits
// 16+4m (little-endian dwords).
void reorder_codes(const uint8_t* qs, uint8_t* out) {
  uint8_t q[32];
  for (int j = 0; j < 16; ++j) {
    q[j] = qs[j] & 15;
    q[j + 16] = qs[j] >> 4;
  }
  for (int i = 0; i < 4; ++i) {
    uint32_t w = 0;
    for (int m = 0; m < 4; ++m) {
      w |= (uint32_t)q[8 * i + 2 * m] << (4 * m);
      w |= (uint32_t)q[8 * i + 2 * m + 1] << (16 + 4 * m);
    }
    memcpy(out + 4 * i, &w, 4);
  }
}

// Source row r (or nullptr for a zero row) of a canonical Q4_0 matrix.
template <typename RowFn>
void pack_gemm_tiles(RowFn row_ptr, int64_t n, int64_t k, uint8_t* out) {
  const int64_t n_tiles = round_up(n, mzk::kGemmTileN) / mzk::kGemmTileN;
  const int64_t k_tiles = round_up(k, mzk::kGemmTileK) / mzk::kGemmTileK;
  const int64_t nb_src = (k + 31) / 32;
  for (int64_t nt = 0; nt < n_tiles; ++nt)
    for (int64_t kt = 0; kt < k_tiles; ++kt) {
      uint8_t* tile = out + (nt * k_tiles + kt) * mzk::kGemmTileBytes;
      for (int r = 0; r < mzk::kGemmTileN; ++r)
        for (int b = 0; b < 2; ++b) {
          const int64_t row = nt * mzk::kGemmTileN + r;
          const int64_t blk = kt * 2 + b;
          uint8_t* nib = tile + (r * 2 + b) * 16;
          uint8_t* sc = tile + mzk::kGemmTileN * mzk::kGemmTileK / 2 + (r * 2 + b) * 2;
          const uint8_t* src = row < n ? row_ptr(row) : nullptr;
          if (src && blk < nb_src) {
            memcpy(sc, src + blk * kBlockBytes, 2);
            reorder_codes(src + blk * kBlockBytes + 2, nib);
          } else {
            memset(sc, 0, 2);          // scale 0: the padded block decodes to 0
            memset(nib, 0x88, 16);
          }
        }
    }
}

void pack_plain(const uint8_t* w, int64_t n, int64_t k, uint8_t* out) {
  const int64_t rb = q4_row_bytes(k);
  pack_gemm_tiles([&](int64_t r) { return w + r * rb; }, n, k, out);
}

// Gate/up interleave: packed row 32 g + i is gate row 16 g + i (i < 16) or up
// row 16 g + i - 16, so a 32-column group of the product holds matching
// gate and up columns.  Each matrix is padded to a multiple of 128 rows.
void pack_gateup(const uint8_t* g, const uint8_t* u, int64_t n, int64_t k, uint8_t* out) {
  const int64_t rb = q4_row_bytes(k);
  const int64_t n_pad = round_up(n, mzk::kGemmTileN / 2);
  pack_gemm_tiles(
      [&](int64_t pr) -> const uint8_t* {
        const int64_t grp = pr / 32, i = pr % 32;
        const int64_t src = grp * 16 + (i < 16 ? i : i - 16);
        if (src >= n) return nullptr;
        return (i < 16 ? g : u) + src * rb;
      },
      2 * n_pad, k, out);
}

// Split rows of 18-byte blocks into nibbles [rows][cols/2] and scales [rows][cols/32].
void split_rows(const uint8_t* w, int64_t rows, int64_t cols, uint8_t* nib, uint16_t* sc) {
  const int64_t nb = cols / 32;
  for (int64_t r = 0; r < rows; ++r)
    for (int64_t b = 0; b < nb; ++b) {
      const uint8_t* blk = w + (r * nb + b) * kBlockBytes;
      memcpy(&sc[r * nb + b], blk, 2);
      memcpy(nib + r * (cols / 2) + b * 16, blk + 2, 16);
    }
}

// ---------------------------------------------------------------- restore rows

struct Rows {
  std::vector<int32_t> nR, nD;
  std::vector<std::vector<int32_t>> R;   // ascending positions per layer
};

// fn(l) for l in [0, L): on host threads when the work (rows to produce) is
// large enough to repay starting them, else in this thread.  fn must only
// touch data of its own layer.
template <class F>
void for_layers(int L, int64_t work, F&& fn) {
  constexpr int64_t kMinWork = 1 << 16;
  const int hw = (int)std::thread::hardware_concurrency();
  const int T = std::min({L, 8, std::max(hw, 1)});
  if (work < kMinWork || T < 2) {
    for (int l = 0; l < L; ++l) fn(l);
    return;
  }
  std::vector<std::exception_ptr> err(T);
  auto run = [&](int t) {
    try {
      for (int l = t; l < L; l += T) fn(l);
    } catch (...) {
      err[t] = std::current_exception();
    }
  };
  std::vector<std::thread> th;
  th.reserve(T - 1);
  for (int t = 1; t < T; ++t) th.emplace_back(run, t);
  run(0);
  for (auto& x : th) x.join();
  for (auto& e : err)
    if (e) std::rethrow_exception(e);
}

// R_l = {p < N : chunk(p) dropped at some l' >= l} U {N..S-1} U {S-1};
// D_l = {p < N : chunk(p) dropped at l} U {N..S-1}.
// Fills `rows`, reusing the capacity of its vectors (a restore's lists are
// megabytes: fresh allocations would fault their pages in on every call).
void compute_rows_into(Rows& rows, const uint8_t* kv_state, int L, int nc, int N, int P, int C) {
  const int S = N + P;
  std::vector<int> maxdrop(nc, -1);
  for (int l = 0; l < L; ++l)
    for (int c = 0; c < nc; ++c)
      if (kv_state[(size_t)l * nc + c] == MZ_DROP) maxdrop[c] = l;
  rows.R.resize(L);
  rows.nR.resize(L);
  rows.nD.resize(L);
  // walked by chunk: the cost is the rows produced, not the cached context
  // (a decode step carries one row per layer of a 32K context); each layer's
  // list is sized first and filled by whole chunk runs
  int64_t total = 0;
  for (int l = 0; l < L; ++l) {
    int nd = P;
    int64_t n = S - N;
    for (int c = 0; c < nc; ++c) {
      const int p0 = c * C, p1 = std::min(N, p0 + C);
      if (maxdrop[c] >= l) n += p1 - p0;
      if (kv_state[(size_t)l * nc + c] == MZ_DROP) nd += p1 - p0;
    }
    const bool last_extra = P == 0 && (N == 0 || maxdrop[nc - 1] < l);   // S - 1 not among the rows yet
    rows.nR[l] = (int32_t)(n + (last_extra ? 1 : 0));
    rows.nD[l] = nd;
    total += rows.nR[l];
  }
  for_layers(L, total, [&](int l) {
    std::vector<int32_t>& r = rows.R[l];
    r.resize((size_t)rows.nR[l]);
    int32_t* o = r.data();
    for (int c = 0; c < nc; ++c) {
      if (maxdrop[c] < l) continue;
      const int p0 = c * C, p1 = std::min(N, p0 + C);
      for (int p = p0; p < p1; ++p) *o++ = p;
    }
    for (int p = N; p < S; ++p) *o++ = p;
    if (o != r.data() + r.size()) *o++ = S - 1;
  });
}

Rows compute_rows(const uint8_t* kv_state, int L, int nc, int N, int P, int C) {
  Rows rows;
  compute_rows_into(rows, kv_state, L, nc, N, P, C);
  return rows;
}

// ---------------------------------------------------------------- pools

struct SlotPool {
  int n = 0;
  int limit = -1;   // test hook: at most this many slots in use (-1: the whole pool)
  std::set<int> free;
  void init(int count) {
    n = count;
    free.clear();
    for (int i = 0; i < count; ++i) free.insert(i);
  }
  int alloc_one() {
    if (free.empty() || (limit >= 0 && used() >= limit)) return -1;
    int s = *free.begin();
    free.erase(free.begin());
    return s;
  }
  // first-fit contiguous run of k slots; -1 if none
  int alloc_run(int k) {
    if (k <= 0 || (limit >= 0 && used() + k > limit)) return -1;
    int start = -1, len = 0, prev = -2;
    for (int s : free) {
      if (s == prev + 1) {
        ++len;
      } else {
        start = s;
        len = 1;
      }
      prev = s;
      if (len == k) {
        for (int i = 0; i < k; ++i) free.erase(start + i);
        return start;
      }
    }
    return -1;
  }
  void release(int s) { free.insert(s); }
  int used() const { return n - (int)free.size(); }
};

struct ArenaEntry {
  int seg;
  size_t off, bytes;
};

// LIFO stack of pinned host segments (the swap space).
struct HostArena {
  struct Seg {
    uint8_t* p;
    size_t cap, used;
  };
  std::vector<Seg> segs;
  int top = 0;
  size_t seg_min = size_t(256) << 20;
  size_t bytes_live = 0;

  uint8_t* ptr(const ArenaEntry& e) const { return segs[e.seg].p + e.off; }

  ArenaEntry push(size_t bytes) {
    bytes = (size_t)round_up((int64_t)bytes, 256);
    while (true) {
      if (top < (int)segs.size() && segs[top].cap - segs[top].used >= bytes) {
        ArenaEntry e{top, segs[top].used, bytes};
        segs[top].used += bytes;
        bytes_live += bytes;
        return e;
      }
      if (top < (int)segs.size() && segs[top].used > 0) {
        ++top;
        continue;
      }
      if (top < (int)segs.size()) {   // empty but too small: replace
        HIPCHK(hipHostFree(segs[top].p));
        segs.erase(segs.begin() + top);
      }
      const size_t cap = std::max(seg_min, bytes);
      void* p = nullptr;
      if (hipHostMalloc(&p, cap, hipHostMallocDefault) != hipSuccess || !p)
        fail(MZ_ENOMEM, "pinned host allocation of %zu bytes failed", cap);
      segs.insert(segs.begin() + std::min<size_t>(top, segs.size()), Seg{(uint8_t*)p, cap, 0});
    }
  }
  void reset() {
    for (auto& s : segs) s.used = 0;
    top = 0;
    bytes_live = 0;
  }
  size_t reserved() const {
    size_t t = 0;
    for (auto& s : segs) t += s.cap;
    return t;
  }
  void release_all() {
    for (auto& s : segs) (void)hipHostFree(s.p);
    segs.clear();
    top = 0;
  }
  // after a restore has consumed the stack: give every segment back
  void trim() {
    for (auto& s : segs)
      if (s.used) fail(MZ_ESTATE, "swap segment still in use");
    for (auto& s : segs) HIPCHK(hipHostFree(s.p));
    segs.clear();
    top = 0;
    bytes_live = 0;
  }
};

// ---------------------------------------------------------------- timing

enum KernelKind {
  kKEmbed, kKRmsnorm, kKGemmKV, kKRopeKV, kKGemmQ, kKRopeQ, kKGather, kKAttention, kKGemmO,
  kKGemmGateUp, kKGemmDown, kKLmHead, kKAttentionSplit, kKGemmQKV1, kKCount
};
const char* kKindName[kKCount] = {"embed_q4", "rmsnorm", "gemm_q4_kv", "rope_kv", "gemm_q4_q",
                                  "rope_q", "gather_rows", "attention", "gemm_q4_o",
                                  "gemm_q4_gateup", "gemm_q4_down", "lm_head_argmax", "attention_split",
                                  "gemm_q4_qkv_one_row"};
// HIP kernel symbol each kind launches (to line up with profiler summaries;
// the Q and K/V projections name their unsplit RoPE-epilogue form)
const char* kKindKernel[kKCount] = {"embed_kernel", "rmsnorm_kernel", "gemm_q4_kernel<5>",
                                    "rope_kv_kernel", "gemm_q4_kernel<4>", "rope_kv_kernel",
                                    "gather_rows_kernel", "attn_kernel", "gemm_q4_kernel<1>",
                                    "gemm_q4_kernel<2>", "gemm_q4_kernel<1>",
                                    "lm_head_kernel+argmax_kernel",
                                    "attn_kernel<split>|attn_few_kernel+attn_merge_wide_kernel",
                                    "gemv1_qkv_kernel"};

struct KindStats {
  int64_t launches = 0;
  double ms = 0, flops = 0, bytes = 0;
};

struct PendingTiming {
  int kind;
  hipEvent_t a, b;
  double flops, bytes;
};

}  // namespace

// ---------------------------------------------------------------- context

struct mz_ctx {
  mz_model_cfg cfg{};
  int device = 0;
  std::string err;
  hipStream_t s_compute = nullptr, s_swap = nullptr;

  // shapes
  int L = 0, d = 0, nq = 0, nkv = 0, hd = 0, ff = 0, ffp = 0, V = 0, C = 0, max_ctx = 0;
  int dq = 0, dkv = 0, dq_pad = 0, kv_pad = 0, d_pad = 0;
  int max_chunks = 0;
  int64_t slot_bytes = 0;
  int64_t off_q = 0, off_kv = 0, off_o = 0, off_gu = 0, off_dn = 0, unit_bytes = 0;

  // weights
  uint8_t* w_slab = nullptr;
  SlotPool w_pool;
  std::vector<int> w_slot;              // per layer, -1 when evicted
  std::vector<uint8_t> w_state;
  std::vector<ArenaEntry> w_entry;
  uint8_t* w_image = nullptr;           // pinned host copy of all packed units
  uint8_t *emb_nib = nullptr, *lm_nib = nullptr;
  uint16_t *emb_sc = nullptr, *lm_sc = nullptr;
  float2* rope_cs = nullptr;

  // KV
  uint8_t* kv_slab = nullptr;
  SlotPool kv_pool;
  std::vector<int32_t> table;           // [L][max_chunks]
  std::vector<uint8_t> kv_state;        // [L][max_chunks]
  std::vector<ArenaEntry> kv_entry;     // [L][max_chunks]
  HostArena arena;

  // context
  std::vector<int32_t> tokens;
  bool have_last = false;
  const float* h_last = nullptr;

  // activations
  float* h[2] = {nullptr, nullptr};
  void* xb = nullptr;      // f16 [max_ctx][max(d, dq)]: norm output / attention output
  float* qf = nullptr;     // [max_ctx][dq_pad]: query projection
  float* kvf = nullptr;    // [max_ctx][kv_pad]: key and value projections
  void* q16 = nullptr;     // f16 [max_ctx][dq]
  void* act = nullptr;     // f16 [max_ctx][ffp]
  float* logits = nullptr;
  float* part_val = nullptr;
  int32_t* part_idx = nullptr;
  int32_t* d_token = nullptr;
  int32_t* d_gen = nullptr;          // [max_ctx] tokens chosen by the steps of mz_generate

  // restore metadata: a pinned staging block and its device mirror of the
  // same size, uploaded by one copy per restore; the pointers below are set
  // per restore to their stretches of the mirror
  uint8_t* d_meta = nullptr;
  int32_t* d_tables = nullptr;
  // per layer: rows whose K/V are written (positions, slot offsets, indices
  // into the layer's input rows) and rows carried on (positions, indices)
  int32_t* d_pos = nullptr;
  int64_t* d_kvoff = nullptr;
  int32_t* d_dix = nullptr;
  int32_t* d_posq = nullptr;
  int32_t* d_qix = nullptr;
  int32_t* d_tok = nullptr;
  uint8_t* h_stage = nullptr;
  size_t stage_bytes = 0;
  int32_t* h_token = nullptr;

  // events
  std::vector<hipEvent_t> ev_w, ev_kv;
  hipEvent_t ev_swap_start = nullptr, ev_swap_end = nullptr;
  bool swap_timed = false;

  // options / stats
  bool overlap = true;
  bool swap_trim = false;               // option swap_trim: free the swap segments after a restore
  int64_t debug_swap_delay_us = 0;   // test hook: delay the swap stream before its copies
  bool debug_poison = false;         // test hook: NaN-fill every freshly allocated unit
  // 8-bit codec on the swap path (option kv_codec): full chunks are compressed
  // into a device staging ring before the copy to host and decompressed from
  // it after the copy back
  bool kv_codec = false;
  int64_t comp_bytes = 0;            // compressed size of one chunk
  uint8_t* codec_stage = nullptr;    // [max_chunks][comp_bytes]
  // partials of split-key attention and split-K GEMMs (few rows: the
  // kernels of one layer run in order on the compute stream and share it)
  uint8_t* split_ws = nullptr;
  int64_t split_ws_bytes = 0;
  bool attn_split = true;            // option attn_split
  // work queues of the persistent attention (zero between launches; the
  // launches run in order on the compute stream)
  int32_t* attn_wq = nullptr;
  bool attn_queue = true;            // option attn_queue
  int32_t* gemm_wq = nullptr;        // the same for the unsplit projections
  bool gemm_queue = true;            // option gemm_queue
  bool gemm_split = true;            // option gemm_split
  bool gemv_direct = true;           // option gemv_direct
  bool gemv_qkv = true;              // option gemv_qkv
  bool fuse_rope = true;             // option fuse_rope: RoPE (and the KV slot writes) in the GEMM epilogue
  bool fuse_norm = true;             // option fuse_norm: a single row's RMSNorm inside its split-K GEMVs

  // Y = X W^T on the compute stream, split over K when the tile grid alone
  // would leave most of the GPU idle.  hn: X is RMSNorm(hn) formed inside the
  // product (only where norm_in_gemv(m, n, k)).
  void gemm(const void* X, int m, int n, int k, const uint8_t* W, int epi, void* Y, hipStream_t s,
            const int32_t* rows = nullptr, const float* hn = nullptr) {
    if (gemv_one(m, n, k)) {
      mzk::launch_gemv1(X, n, k, W, epi, mzk::GemmRope{}, Y, s, rows, hn, cfg.rms_eps);
      return;
    }
    const int ns = gemm_split ? mzk::gemm_auto_splits(m, n, k, split_ws_bytes) : 1;
    if (ns > 1)
      mzk::launch_gemm_q4_splitk(X, m, n, k, W, epi, Y, ns, split_ws, s, rows, hn, cfg.rms_eps);
    else
      mzk::launch_gemm_q4(X, m, n, k, W, epi, Y, s, rows, gemm_queue ? gemm_wq : nullptr,
                          gemm_split ? split_ws : nullptr, split_ws_bytes);
  }
  // The projection with rotary embedding fused into its epilogue (or into
  // the reduce of its K splits), when the shape allows it (false: the caller
  // runs the projection and the RoPE kernel separately).
  bool gemm_rope(const void* X, int m, int n, int k, const uint8_t* W, int epi, const mzk::GemmRope& ea, void* Y,
                 hipStream_t s, const int32_t* rows, const float* hn = nullptr) {
    if (!fuse_rope || !mzk::gemm_rope_fusable(ea.hd, ea.C)) return false;
    if (gemv_one(m, n, k)) {
      mzk::launch_gemv1(X, n, k, W, epi, ea, Y, s, rows, hn, cfg.rms_eps);
      return true;
    }
    const int ns = gemm_split ? mzk::gemm_auto_splits(m, n, k, split_ws_bytes) : 1;
    if (ns > 1)
      mzk::launch_gemm_q4_splitk_rope(X, m, n, k, W, epi, ea, Y, ns, split_ws, s, rows, hn, cfg.rms_eps);
    else
      mzk::launch_gemm_q4_rope(X, m, n, k, W, epi, ea, Y, s, rows, nullptr, gemm_split ? split_ws : nullptr,
                               split_ws_bytes);
    return true;
  }
  // A one-row product that runs as the split-K GEMV, which can normalize its
  // own input row (a decode step: the RMSNorm launch is then left out)
  bool norm_in_gemv(int m, int n, int k) const {
    return fuse_norm && m == 1 &&
           (gemv_one(m, n, k) || (gemm_split && mzk::gemm_auto_splits(m, n, k, split_ws_bytes) > 1));
  }
  // An unsplit attention launch takes the work queues (option attn_queue)
  // from 4 (query tile, KV head) items per CU on; a workgroup covers 256
  // (query row, query head) pairs.  The queues even out XCDs that run at
  // different clocks, which takes several rounds of items; with fewer, one
  // workgroup per item is as fast or faster, with the same results.
  // Measured on one MI355X, persistent against one item per workgroup, causal rows:
  // 2048 rows, 32/8 heads of 64 (256 items): 55.2 against 41.4 us; 8256
  // rows, 24/8 heads of 128 (792): 449 against 446; 8320 rows, 32/8 heads of
  // 128 (1040): 548 against 558; 32896 rows (4112): 7890 against 8200.
  bool attn_queue_pays(int m) const {
    static const int cus = [] {
      int dev = 0, n = 0;
      if (hipGetDevice(&dev) != hipSuccess ||
          hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
        n = 256;
      return n;
    }();
    constexpr int64_t kMinItemsPerCu = 4, kPairsPerItem = 256;
    return attn_queue && (int64_t)m * nq >= kMinItemsPerCu * kPairsPerItem * cus;
  }
  // A single row runs as the one-launch GEMV (option gemv_direct)
  bool gemv_one(int m, int n, int k) const { return gemv_direct && m == 1 && mzk::gemv1_ok(n, k); }
  int32_t* d_codec_slots = nullptr;  // per restore: destination slot of each compressed chunk (in d_meta)
  hipEvent_t ev_meta = nullptr;      // restore metadata uploaded (the swap stream reads some)
  bool meta_recorded = false;        // ev_meta stands for an upload from the staging block
  bool timing = false;
  std::vector<hipEvent_t> ev_pool;
  size_t ev_used = 0;
  std::vector<PendingTiming> pending;
  KindStats kstats[kKCount];
  std::vector<int32_t> last_nR, last_nD, last_nQ;
  Rows rows_buf;                     // row lists of the last restore (capacity kept)
  int64_t last_swap_kv_bytes = 0, last_swap_w_bytes = 0, last_reload_w_bytes = 0;
  int64_t last_copies = 0;
  double last_swap_ms = -1;
  double last_algo_flops = 0;
  // host time of the last restore: planning + metadata staging until the
  // first kernel is queued, and the whole call (everything queued)
  double last_plan_ms = 0, last_enqueue_ms = 0;
  int last_N = 0, last_P = 0;

  hipEvent_t get_event() {
    if (ev_used == ev_pool.size()) {
      hipEvent_t e;
      HIPCHK(hipEventCreate(&e));
      ev_pool.push_back(e);
    }
    return ev_pool[ev_used++];
  }

  template <typename F>
  void timed(int kind, double flops, double bytes, hipStream_t s, F&& launch) {
    if (!timing) {
      launch();
      HIPCHK(hipGetLastError());
      return;
    }
    hipEvent_t a = get_event(), b = get_event();
    HIPCHK(hipEventRecord(a, s));
    launch();
    HIPCHK(hipGetLastError());
    HIPCHK(hipEventRecord(b, s));
    pending.push_back({kind, a, b, flops, bytes});
  }

  void collect_timing() {
    for (auto& p : pending) {
      float ms = 0;
      HIPCHK(hipEventElapsedTime(&ms, p.a, p.b));
      KindStats& k = kstats[p.kind];
      k.launches++;
      k.ms += ms;
      k.flops += p.flops;
      k.bytes += p.bytes;
    }
    pending.clear();
    ev_used = 0;
  }

  uint8_t* unit_ptr(int l) const { return w_slab + (int64_t)w_slot[l] * unit_bytes; }
  int nchunks_of(int n_tokens) const { return (n_tokens + C - 1) / C; }

  void release_context() {
    // the arena is cleared below: swapped weight units come back from the image
    for (int l = 0; l < L; ++l)
      if (w_state[l] == MZ_SWAP) w_state[l] = MZ_DROP;
    for (int l = 0; l < L; ++l)
      for (int c = 0; c < max_chunks; ++c) {
        int32_t& t = table[(size_t)l * max_chunks + c];
        if (t >= 0) kv_pool.release(t);
        t = -1;
        kv_state[(size_t)l * max_chunks + c] = MZ_RES;
      }
    arena.reset();
    tokens.clear();
    have_last = false;
  }
};

namespace {

template <typename F>
mz_status guarded(mz_ctx* ctx, F&& body) {
  try {
    if (ctx) {
      ctx->err.clear();
      HIPCHK(hipSetDevice(ctx->device));
    }
    body();
    return MZ_OK;
  } catch (const StatusError& e) {
    if (ctx) ctx->err = e.msg; else g_load_error = e.msg;
    return e.st;
  } catch (const HipError& e) {
    std::string m = std::string("HIP error '") + hipGetErrorString(e.e) + "' in " + e.what;
    if (ctx) ctx->err = m; else g_load_error = m;
    return MZ_EHIP;
  } catch (const std::bad_alloc&) {
    if (ctx) ctx->err = "host allocation failed"; else g_load_error = "host allocation failed";
    return MZ_ENOMEM;
  }
}

void* dmalloc(size_t bytes) {
  void* p = nullptr;
  if (hipMalloc(&p, std::max<size_t>(bytes, 256)) != hipSuccess || !p)
    fail(MZ_ENOMEM, "device allocation of %zu bytes failed", bytes);
  return p;
}

void validate_cfg(const mz_model_cfg* c) {
  if (!c) fail(MZ_EINVAL, "cfg is NULL");
  if (c->n_layers < 1 || c->d_model < 256 || c->d_model % 256 || c->d_model > 8192)
    fail(MZ_EINVAL, "d_model must be a multiple of 256 in 256..8192 and n_layers >= 1");
  if (c->head_dim != 64 && c->head_dim != 128) fail(MZ_EINVAL, "head_dim must be 64 or 128");
  if (c->n_kv_heads < 1 || c->n_q_heads < 1 || c->n_q_heads % c->n_kv_heads)
    fail(MZ_EINVAL, "n_q_heads must be a positive multiple of n_kv_heads");
  if (c->n_q_heads / c->n_kv_heads > 8) fail(MZ_EINVAL, "GQA group above 8 is not supported");
  if (c->d_ffn < 1 || c->vocab < 1) fail(MZ_EINVAL, "d_ffn and vocab must be positive");
  if (c->chunk_tokens < 8 || (c->chunk_tokens & (c->chunk_tokens - 1)) || c->max_ctx < 1)
    fail(MZ_EINVAL, "chunk_tokens must be a power of two >= 8 and max_ctx positive");
  if ((c->max_ctx + c->chunk_tokens - 1) / c->chunk_tokens > mzk::kAttnTableMax)
    fail(MZ_EINVAL, "max_ctx / chunk_tokens exceeds %d chunks per layer", mzk::kAttnTableMax);
  if (!(c->rope_theta > 0) || !(c->rms_eps >= 0)) fail(MZ_EINVAL, "rope_theta must be > 0 and rms_eps >= 0");
}

int64_t blob_bytes(const mz_model_cfg* c) {
  const int64_t d = c->d_model, dq = (int64_t)c->n_q_heads * c->head_dim,
                dkv = (int64_t)c->n_kv_heads * c->head_dim, ff = c->d_ffn;
  const int64_t layer = dq * q4_row_bytes(d) + 2 * dkv * q4_row_bytes(d) + d * q4_row_bytes(dq) +
                        2 * ff * q4_row_bytes(d) + d * q4_row_bytes(ff);
  return c->n_layers * layer + 2 * (int64_t)c->vocab * q4_row_bytes(d);
}

}  // namespace

namespace mzrt {
int64_t weight_unit_bytes(const mz_model_cfg& cfg) { return unit_layout(cfg).unit_bytes; }
int64_t kv_slot_bytes(const mz_model_cfg& cfg) {
  return (int64_t)cfg.chunk_tokens * cfg.n_kv_heads * cfg.head_dim * 2 * 2;
}
void set_error(const char* msg) { g_load_error = msg; }
}  // namespace mzrt

// ---------------------------------------------------------------- restore core

namespace {

struct CopyJob {
  void* dst;
  const void* src;
  size_t bytes;
};

// Shared by mz_restore_and_prefill and mz_prefill_context.
// dev_tok (device, or null): the last prompt token is read from there by the
// embedding instead of from prompt (a decode step whose token the previous
// step left on the device; prompt then holds a placeholder).
void restore_and_prefill_impl(mz_ctx* x, const int32_t* prompt, int32_t n_prompt,
                              const int32_t* dev_tok = nullptr) {
  const auto t_entry = std::chrono::steady_clock::now();
  auto ms_since = [&](std::chrono::steady_clock::time_point t) {
    return std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t).count();
  };
  const int L = x->L, C = x->C, MC = x->max_chunks;
  if (n_prompt < 0) fail(MZ_EINVAL, "n_prompt is negative");
  if (n_prompt > 0 && !prompt) fail(MZ_EINVAL, "prompt is NULL");
  const int N = (int)x->tokens.size();
  const int P = n_prompt;
  const int S = N + P;
  if (S == 0) fail(MZ_ESTATE, "no context and no prompt to prefill");
  if (S > x->max_ctx) fail(MZ_EINVAL, "context + prompt (%d) exceeds max_ctx (%d)", S, x->max_ctx);
  for (int i = 0; i < P; ++i)
    if (prompt[i] < 0 || prompt[i] >= x->V) fail(MZ_EINVAL, "prompt token %d out of range", prompt[i]);
  const int nc_old = x->nchunks_of(N), nc_new = x->nchunks_of(S);

  // --- plan rows over the chunks of the cached context
  std::vector<uint8_t> st((size_t)L * std::max(nc_old, 1), MZ_RES);
  for (int l = 0; l < L; ++l)
    for (int c = 0; c < nc_old; ++c) st[(size_t)l * nc_old + c] = x->kv_state[(size_t)l * MC + c];
  Rows& rows = x->rows_buf;
  compute_rows_into(rows, st.data(), L, nc_old, N, P, C);

  // --- allocate slots: swapped chunks first, in runs matching their arena order
  std::vector<std::vector<CopyJob>> kv_jobs(L);
  // compressed chunks: copies of arena runs into the staging ring (in the
  // layer's compressed order) and the slot each one decompresses into
  std::vector<std::vector<CopyJob>> codec_jobs(L);
  std::vector<std::vector<int32_t>> codec_slots(L);
  std::vector<int> new_slots;   // for rollback on failure
  auto rollback = [&]() {
    for (int s : new_slots) x->kv_pool.release(s);
  };
  try {
    for (int l = 0; l < L; ++l) {
      std::vector<int> sw, swc;
      for (int c = 0; c < nc_old; ++c)
        if (x->kv_state[(size_t)l * MC + c] == MZ_SWAP)
          (x->kv_entry[(size_t)l * MC + c].bytes == (size_t)x->slot_bytes ? sw : swc).push_back(c);
      auto by_arena = [&](int a, int b) {
        const ArenaEntry &ea = x->kv_entry[(size_t)l * MC + a], &eb = x->kv_entry[(size_t)l * MC + b];
        return ea.seg != eb.seg ? ea.seg < eb.seg : ea.off < eb.off;
      };
      std::sort(swc.begin(), swc.end(), by_arena);
      for (size_t i = 0; i < swc.size();) {
        size_t j = i + 1;
        while (j < swc.size()) {
          const ArenaEntry &p = x->kv_entry[(size_t)l * MC + swc[j - 1]], &q = x->kv_entry[(size_t)l * MC + swc[j]];
          if (q.seg != p.seg || q.off != p.off + p.bytes) break;
          ++j;
        }
        codec_jobs[l].push_back({x->codec_stage + (int64_t)i * x->comp_bytes,
                                 x->arena.ptr(x->kv_entry[(size_t)l * MC + swc[i]]),
                                 (size_t)(j - i) * (size_t)x->comp_bytes});
        i = j;
      }
      for (int c : swc) {
        const int sl = x->kv_pool.alloc_one();
        if (sl < 0) fail(MZ_ENOMEM, "KV slot pool exhausted");
        x->table[(size_t)l * MC + c] = sl;
        new_slots.push_back(sl);
        codec_slots[l].push_back(sl);
      }
      std::sort(sw.begin(), sw.end(), by_arena);
      size_t i = 0;
      while (i < sw.size()) {
        size_t j = i + 1;
        while (j < sw.size()) {
          const ArenaEntry &p = x->kv_entry[(size_t)l * MC + sw[j - 1]], &q = x->kv_entry[(size_t)l * MC + sw[j]];
          if (q.seg != p.seg || q.off != p.off + p.bytes) break;
          ++j;
        }
        // arena run sw[i..j): try one contiguous slot run, else split per chunk
        const int k = (int)(j - i);
        int first = x->kv_pool.alloc_run(k);
        if (first >= 0) {
          for (int t = 0; t < k; ++t) {
            x->table[(size_t)l * MC + sw[i + t]] = first + t;
            new_slots.push_back(first + t);
          }
          const ArenaEntry& e0 = x->kv_entry[(size_t)l * MC + sw[i]];
          kv_jobs[l].push_back({x->kv_slab + (int64_t)first * x->slot_bytes, x->arena.ptr(e0),
                                (size_t)k * (size_t)x->slot_bytes});
        } else {
          for (int t = 0; t < k; ++t) {
            int s = x->kv_pool.alloc_one();
            if (s < 0) fail(MZ_ENOMEM, "KV slot pool exhausted");
            x->table[(size_t)l * MC + sw[i + t]] = s;
            new_slots.push_back(s);
            const ArenaEntry& e = x->kv_entry[(size_t)l * MC + sw[i + t]];
            kv_jobs[l].push_back({x->kv_slab + (int64_t)s * x->slot_bytes, x->arena.ptr(e),
                                  (size_t)x->slot_bytes});
          }
        }
        i = j;
      }
    }
    for (int l = 0; l < L; ++l) {
      for (int c = 0; c < nc_new; ++c) {
        int32_t& t = x->table[(size_t)l * MC + c];
        const bool need = c >= nc_old || x->kv_state[(size_t)l * MC + c] == MZ_DROP;
        if (need && t < 0) {
          int s = x->kv_pool.alloc_one();
          if (s < 0) fail(MZ_ENOMEM, "KV slot pool exhausted");
          t = s;
          new_slots.push_back(s);
        }
      }
    }
  } catch (...) {
    for (int l = 0; l < L; ++l)
      for (int c = 0; c < MC; ++c) {
        int32_t& t = x->table[(size_t)l * MC + c];
        if (t >= 0 && std::find(new_slots.begin(), new_slots.end(), t) != new_slots.end()) t = -1;
      }
    rollback();
    throw;
  }
  // weight units
  std::vector<int> w_new;
  for (int l = 0; l < L; ++l)
    if (x->w_state[l] != MZ_RES) {
      int s = x->w_pool.alloc_one();
      if (s < 0) fail(MZ_ENOMEM, "weight unit pool exhausted");
      x->w_slot[l] = s;
      w_new.push_back(l);
    }

  // --- metadata: tables; per layer the rows whose K/V are written (D_l:
  // position, slot offset, index among the layer's input rows R_l) and the
  // rows carried on (R_{l+1}, or the last position after the last layer:
  // position, index in R_l); tokens
  std::vector<int64_t> dofs(L + 1, 0), qofs(L + 1, 0), cofs(L + 1, 0);
  for (int l = 0; l < L; ++l) cofs[l + 1] = cofs[l] + (int64_t)codec_slots[l].size();
  std::vector<int32_t> nQ(L);
  for (int l = 0; l < L; ++l) {
    nQ[l] = l + 1 < L ? rows.nR[l + 1] : 1;
    dofs[l + 1] = dofs[l] + rows.nD[l];
    qofs[l + 1] = qofs[l] + nQ[l];
  }
  const size_t b_tab = (size_t)L * MC * 4, b_pos = (size_t)dofs[L] * 4, b_off = (size_t)dofs[L] * 8,
               b_dix = (size_t)dofs[L] * 4, b_posq = (size_t)qofs[L] * 4, b_qix = (size_t)qofs[L] * 4,
               b_tok = (size_t)rows.nR[0] * 4, b_cs = (size_t)cofs[L] * 4;
  const size_t need = b_tab + b_pos + b_off + b_dix + b_posq + b_qix + b_tok + b_cs + 8 * 256;
  if (need > x->stage_bytes) fail(MZ_EINVAL, "restore metadata exceeds the staging buffer");
  // the staging block is rewritten only after the previous restore's upload
  // out of it has been done (a restore issued before the last one's first
  // token may find it still in flight)
  if (x->meta_recorded) HIPCHK(hipEventSynchronize(x->ev_meta));
  uint8_t* sp = x->h_stage;
  int32_t* s_tab = (int32_t*)sp;
  int32_t* s_pos = (int32_t*)(sp + round_up(b_tab, 256));
  int64_t* s_off = (int64_t*)((uint8_t*)s_pos + round_up(b_pos, 256));
  int32_t* s_dix = (int32_t*)((uint8_t*)s_off + round_up(b_off, 256));
  int32_t* s_posq = (int32_t*)((uint8_t*)s_dix + round_up(b_dix, 256));
  int32_t* s_qix = (int32_t*)((uint8_t*)s_posq + round_up(b_posq, 256));
  int32_t* s_tok = (int32_t*)((uint8_t*)s_qix + round_up(b_qix, 256));
  int32_t* s_cs = (int32_t*)((uint8_t*)s_tok + round_up(b_tok, 256));
  for (int l = 0; l < L; ++l)
    if (!codec_slots[l].empty())
      memcpy(s_cs + cofs[l], codec_slots[l].data(), codec_slots[l].size() * 4);
  memcpy(s_tab, x->table.data(), b_tab);
  int64_t total_rows = 0;
  for (int l = 0; l < L; ++l) total_rows += rows.nR[l];
  std::vector<char> count_ok(L, 1);
  for_layers(L, total_rows, [&](int l) {
    const std::vector<int32_t>& R = rows.R[l];
    int64_t j = dofs[l];
    for (size_t i = 0; i < R.size(); ++i) {
      const int p = R[i];
      const int c = p / C;
      if (p >= N || x->kv_state[(size_t)l * MC + c] == MZ_DROP) {
        s_pos[j] = p;
        s_off[j] = (int64_t)x->table[(size_t)l * MC + c] * x->slot_bytes + (int64_t)(p % C) * x->dkv * 2;
        s_dix[j] = (int32_t)i;
        ++j;
      }
    }
    if (j != dofs[l + 1]) count_ok[l] = 0;
    if (l + 1 < L) {
      const std::vector<int32_t>& Rn = rows.R[l + 1];
      size_t a = 0;
      for (size_t b = 0; b < Rn.size(); ++b) {
        while (R[a] != Rn[b]) ++a;
        s_posq[qofs[l] + b] = Rn[b];
        s_qix[qofs[l] + b] = (int32_t)a;
      }
    } else {
      s_posq[qofs[l]] = R.back();             // S - 1
      s_qix[qofs[l]] = (int32_t)R.size() - 1;
    }
  });
  for (int l = 0; l < L; ++l)
    if (!count_ok[l]) fail(MZ_EINVAL, "internal: written-row count mismatch at layer %d", l);
  for (int i = 0; i < rows.nR[0]; ++i) {
    const int p = rows.R[0][i];
    s_tok[i] = p < N ? x->tokens[p] : prompt[p - N];
  }
  hipStream_t cs = x->s_compute, ss = x->s_swap;
  // one upload of the whole staged stretch: each copy call costs tens of
  // microseconds of host time, which a one-token step waits on in full
  auto dev = [&](const void* hp) { return x->d_meta + ((const uint8_t*)hp - sp); };
  x->d_tables = (int32_t*)dev(s_tab);
  x->d_pos = (int32_t*)dev(s_pos);
  x->d_kvoff = (int64_t*)dev(s_off);
  x->d_dix = (int32_t*)dev(s_dix);
  x->d_posq = (int32_t*)dev(s_posq);
  x->d_qix = (int32_t*)dev(s_qix);
  x->d_tok = (int32_t*)dev(s_tok);
  x->d_codec_slots = (int32_t*)dev(s_cs);
  const size_t b_meta = (size_t)((const uint8_t*)s_cs - sp) + b_cs;
  if (b_meta > x->stage_bytes) fail(MZ_EINVAL, "internal: restore metadata overruns the staging buffer");
  HIPCHK(hipMemcpyAsync(x->d_meta, sp, b_meta, hipMemcpyHostToDevice, cs));
  HIPCHK(hipEventRecord(x->ev_meta, cs));
  x->meta_recorded = true;

  if (x->debug_poison) {
    // fresh slots hold fp16 NaN until restored or recomputed: a missed row or
    // an unordered read shows up as NaN
    std::vector<char> is_copy_dst((size_t)x->kv_pool.n, 0);
    for (int l = 0; l < L; ++l)
      for (int c = 0; c < nc_old; ++c)
        if (x->kv_state[(size_t)l * MC + c] == MZ_SWAP) is_copy_dst[x->table[(size_t)l * MC + c]] = 1;
    for (int sl : new_slots)
      mzk::launch_fill(x->kv_slab + (int64_t)sl * x->slot_bytes, x->slot_bytes / 4, 0xFFFFFFFFu,
                       is_copy_dst[sl] ? ss : cs);
    for (int l : w_new) mzk::launch_fill(x->unit_ptr(l), x->unit_bytes / 4, 0xFFFFFFFFu, ss);
    HIPCHK(hipGetLastError());
  }
  if (x->debug_swap_delay_us > 0) {
    mzk::launch_spin(x->debug_swap_delay_us, ss);
    HIPCHK(hipGetLastError());
  }

  // --- swap-in on the side stream, forward-in, one event per layer and kind
  std::vector<char> w_copy(L, 0), kv_copy(L, 0);
  int64_t swap_kv = 0, swap_w = 0, reload_w = 0, copies = 0;
  x->swap_timed = false;
  bool any_copy = false;
  for (int l = 0; l < L; ++l)
    any_copy |= x->w_state[l] != MZ_RES || !kv_jobs[l].empty() || !codec_jobs[l].empty();
  if (any_copy) {
    HIPCHK(hipEventRecord(x->ev_swap_start, ss));
    if (b_cs) HIPCHK(hipStreamWaitEvent(ss, x->ev_meta, 0));   // slot lists of the decompressions
    for (int l = 0; l < L; ++l) {
      if (x->w_state[l] != MZ_RES) {
        const void* src = x->w_state[l] == MZ_SWAP ? (const void*)x->arena.ptr(x->w_entry[l])
                                                    : (const void*)(x->w_image + (int64_t)l * x->unit_bytes);
        HIPCHK(hipMemcpyAsync(x->unit_ptr(l), src, x->unit_bytes, hipMemcpyHostToDevice, ss));
        HIPCHK(hipEventRecord(x->ev_w[l], ss));
        w_copy[l] = 1;
        (x->w_state[l] == MZ_SWAP ? swap_w : reload_w) += x->unit_bytes;
        ++copies;
      }
      for (const CopyJob& j : kv_jobs[l]) {
        HIPCHK(hipMemcpyAsync(j.dst, j.src, j.bytes, hipMemcpyHostToDevice, ss));
        swap_kv += j.bytes;
        ++copies;
      }
      for (const CopyJob& j : codec_jobs[l]) {
        HIPCHK(hipMemcpyAsync(j.dst, j.src, j.bytes, hipMemcpyHostToDevice, ss));
        swap_kv += j.bytes;
        ++copies;
      }
      if (!codec_slots[l].empty()) {
        mzk::launch_kv_decompress(x->codec_stage, x->slot_bytes / 2, (int)codec_slots[l].size(), x->kv_slab,
                                  x->d_codec_slots + cofs[l], x->slot_bytes, ss);
        HIPCHK(hipGetLastError());
      }
      if (!kv_jobs[l].empty() || !codec_slots[l].empty()) {
        HIPCHK(hipEventRecord(x->ev_kv[l], ss));
        kv_copy[l] = 1;
      }
    }
    HIPCHK(hipEventRecord(x->ev_swap_end, ss));
    x->swap_timed = true;
    if (!x->overlap) HIPCHK(hipStreamWaitEvent(cs, x->ev_swap_end, 0));
  }

  x->last_plan_ms = ms_since(t_entry);
  // --- compute stream: embedding, layers, compaction
  const int d = x->d;
  const double bpe_w = 0.5625;   // Q4_0 bytes per weight
  x->timed(kKEmbed, 0, (double)rows.nR[0] * (d * bpe_w + d * 4.0), cs, [&] {
    mzk::launch_embed(x->emb_nib, x->emb_sc, x->d_tok, rows.nR[0], d, x->h[0], cs, dev_tok);
  });
  int cur = 0;
  double algo = 2.0 * d * x->V;
  for (int l = 0; l < L; ++l) {
    const int n = rows.nR[l], nd = rows.nD[l], nq = nQ[l];
    if (w_copy[l]) HIPCHK(hipStreamWaitEvent(cs, x->ev_w[l], 0));
    const uint8_t* unit = x->unit_ptr(l);
    float* h = x->h[cur];
    // a single row whose projections all run as GEMVs normalizes inside them
    const bool norm1_fused = n == 1 && (nd == 0 || x->norm_in_gemv(nd, x->kv_pad, d)) &&
                             (nq == 0 || x->norm_in_gemv(nq, x->dq_pad, d));
    const float* hn1 = norm1_fused ? h : nullptr;
    if (!norm1_fused)
      x->timed(kKRmsnorm, 0, (double)n * d * 6.0, cs,
               [&] { mzk::launch_rmsnorm(h, n, d, x->cfg.rms_eps, x->xb, cs); });
    // prompt rows appended to a partial last chunk that was swapped out land in
    // the restored slot: its copy must be done before they are written
    const bool early_wait = kv_copy[l] && P > 0 && N % C != 0 &&
                            x->kv_state[(size_t)l * MC + (nc_old - 1)] == MZ_SWAP;
    if (early_wait) HIPCHK(hipStreamWaitEvent(cs, x->ev_kv[l], 0));
    const int32_t* qix = x->d_qix + qofs[l];
    const int32_t* posq = x->d_posq + qofs[l];
    // a single row's query and key/value products in one launch
    const bool qkv1 = x->gemv_qkv && nd == 1 && nq == 1 && x->fuse_rope && mzk::gemm_rope_fusable(x->hd, C) &&
                      x->gemv_one(1, x->kv_pad, d) && x->gemv_one(1, x->dq_pad, d);
    if (qkv1) {
      mzk::GemmRope ekv, eq;
      ekv.pos = x->d_pos + dofs[l];
      ekv.kv_off = x->d_kvoff + dofs[l];
      ekv.rope_cs = x->rope_cs;
      ekv.slab = x->kv_slab;
      ekv.hd = x->hd;
      ekv.n_valid = 2 * x->dkv;
      ekv.C = C;
      eq.pos = posq;
      eq.rope_cs = x->rope_cs;
      eq.hd = x->hd;
      eq.n_valid = x->dq;
      eq.C = C;
      x->timed(kKGemmQKV1, 2.0 * d * (2 * x->dkv + x->dq), (2.0 * x->dkv + x->dq) * d * bpe_w +
                                                              d * 4.0 + (2 * x->dkv + x->dq) * 2.0,
               cs, [&] {
                 mzk::launch_gemv1_qkv(x->xb, d, unit + x->off_q, x->q16, eq, qix, unit + x->off_kv, ekv,
                                       x->d_dix + dofs[l], cs, hn1, x->cfg.rms_eps);
               });
    }
    // keys and values of the rows written at this layer (D_l)
    if (nd > 0 && !qkv1) {
      const int32_t* dix = x->d_dix + dofs[l];
      mzk::GemmRope ea;
      ea.pos = x->d_pos + dofs[l];
      ea.kv_off = x->d_kvoff + dofs[l];
      ea.rope_cs = x->rope_cs;
      ea.slab = x->kv_slab;
      ea.hd = x->hd;
      ea.n_valid = 2 * x->dkv;
      ea.C = C;
      bool fused = false;
      x->timed(kKGemmKV, 2.0 * nd * d * 2 * x->dkv, 2.0 * x->dkv * d * bpe_w + nd * (d * 2.0 + 2 * x->dkv * 2.0), cs,
               [&] {
                 fused = x->gemm_rope(x->xb, nd, x->kv_pad, d, unit + x->off_kv, mzk::kEpiRopeKV, ea, nullptr, cs,
                                      dix, hn1);
                 if (!fused)
                   x->gemm(x->xb, nd, x->kv_pad, d, unit + x->off_kv, mzk::kEpiStore, x->kvf, cs, dix, hn1);
               });
      if (!fused)
        x->timed(kKRopeKV, 0, nd * (2 * x->dkv * 4.0 + 2 * x->dkv * 2.0), cs, [&] {
          mzk::launch_rope_kv(x->kvf, x->kv_pad, nd, x->d_pos + dofs[l], x->d_kvoff + dofs[l], x->rope_cs, 0,
                              x->nkv, x->hd, C, nullptr, x->kv_slab, cs);
        });
    }
    if (kv_copy[l] && !early_wait) HIPCHK(hipStreamWaitEvent(cs, x->ev_kv[l], 0));
    // queries, attention and MLP of the rows carried on (R_{l+1}; the last
    // position after the last layer)
    if (!qkv1) {
      mzk::GemmRope ea;
      ea.pos = posq;
      ea.rope_cs = x->rope_cs;
      ea.hd = x->hd;
      ea.n_valid = x->dq;
      ea.C = C;
      bool fused = false;
      x->timed(kKGemmQ, 2.0 * nq * d * x->dq, (double)x->dq * d * bpe_w + nq * (d * 2.0 + x->dq * 2.0), cs, [&] {
        fused = x->gemm_rope(x->xb, nq, x->dq_pad, d, unit + x->off_q, mzk::kEpiRopeQ, ea, x->q16, cs, qix, hn1);
        if (!fused) x->gemm(x->xb, nq, x->dq_pad, d, unit + x->off_q, mzk::kEpiStore, x->qf, cs, qix, hn1);
      });
      if (!fused)
        x->timed(kKRopeQ, 0, nq * (x->dq * 4.0 + x->dq * 2.0), cs, [&] {
          mzk::launch_rope_kv(x->qf, x->dq_pad, nq, posq, nullptr, x->rope_cs, x->nq, 0, x->hd, C, x->q16,
                              x->kv_slab, cs);
        });
    }
    if (nq < n) {
      float* dst = x->h[cur ^ 1];
      x->timed(kKGather, 0, (double)nq * d * 8.0, cs,
               [&] { mzk::launch_gather_rows(h, qix, nq, d, dst, cs); });
      cur ^= 1;
      h = dst;
    }
    double keys = 0;
    if (l + 1 < L)
      for (int p : rows.R[l + 1]) keys += p + 1.0;
    else
      keys = S;
    const double att_flops = 4.0 * x->hd * x->nq * keys;
    // few query rows against a long context: split the keys over the chip
    const int max_pos = l + 1 < L ? rows.R[l + 1].back() : S - 1;
    const int n_split =
        x->attn_split ? mzk::attention_auto_splits(nq, max_pos, x->nq, x->nkv, x->hd, x->split_ws_bytes) : 1;
    x->timed(n_split > 1 ? kKAttentionSplit : kKAttention, att_flops, (double)nq * x->dq * 4.0, cs, [&] {
      if (n_split > 1)
        mzk::launch_attention_split(x->q16, posq, nq, max_pos, x->kv_slab, x->d_tables + (size_t)l * MC, MC, C,
                                    x->slot_bytes, x->nq, x->nkv, x->hd, n_split, x->split_ws, x->xb, cs);
      else
        mzk::launch_attention(x->q16, posq, nq, x->kv_slab, x->d_tables + (size_t)l * MC, MC, C, x->slot_bytes,
                              x->nq, x->nkv, x->hd, x->xb, cs, x->attn_queue_pays(nq) ? x->attn_wq : nullptr);
    });
    x->timed(kKGemmO, 2.0 * nq * x->dq * d, (double)d * x->dq * bpe_w + nq * (x->dq * 2.0 + d * 8.0), cs,
             [&] { x->gemm(x->xb, nq, x->d_pad, x->dq, unit + x->off_o, mzk::kEpiAdd, h, cs); });
    const float* hn2 = x->norm_in_gemv(nq, 2 * x->ffp, d) ? h : nullptr;
    if (!hn2)
      x->timed(kKRmsnorm, 0, (double)nq * d * 6.0, cs,
               [&] { mzk::launch_rmsnorm(h, nq, d, x->cfg.rms_eps, x->xb, cs); });
    x->timed(kKGemmGateUp, 2.0 * nq * d * 2.0 * x->ff, 2.0 * x->ff * d * bpe_w + nq * (d * 2.0 + x->ff * 2.0), cs,
             [&] { x->gemm(x->xb, nq, 2 * x->ffp, d, unit + x->off_gu, mzk::kEpiSwiGLU, x->act, cs, nullptr, hn2); });
    x->timed(kKGemmDown, 2.0 * nq * x->ff * d, (double)d * x->ff * bpe_w + nq * (x->ffp * 2.0 + d * 8.0), cs,
             [&] { x->gemm(x->act, nq, x->d_pad, x->ffp, unit + x->off_dn, mzk::kEpiAdd, h, cs); });
    algo += 2.0 * nd * d * 2 * x->dkv + 2.0 * nq * d * 2 * x->dq + 2.0 * nq * 3 * d * x->ff + att_flops;
  }
  x->h_last = x->h[cur];
  x->have_last = true;
  x->last_nQ = nQ;

  // --- new state: every unit resident, context extended by the prompt
  for (int l = 0; l < L; ++l) {
    x->w_state[l] = MZ_RES;
    for (int c = 0; c < MC; ++c) x->kv_state[(size_t)l * MC + c] = MZ_RES;
  }
  x->arena.reset();
  if (x->swap_trim) {   // the copies out of the segments must be done before they are freed
    HIPCHK(hipStreamSynchronize(x->s_swap));
    x->arena.trim();
  }
  x->tokens.insert(x->tokens.end(), prompt, prompt + P);
  x->last_nR = rows.nR;
  x->last_nD = rows.nD;
  x->last_swap_kv_bytes = swap_kv;
  x->last_swap_w_bytes = swap_w;
  x->last_reload_w_bytes = reload_w;
  x->last_copies = copies;
  x->last_algo_flops = algo;
  x->last_enqueue_ms = ms_since(t_entry);
  x->last_N = N;
  x->last_P = P;
  x->last_swap_ms = -1;
}

}  // namespace

// ---------------------------------------------------------------- ABI

extern "C" {

const char* mz_version(void) { return kVersion; }

const char* mz_last_error(const mz_ctx* ctx) {
  return ctx ? ctx->err.c_str() : g_load_error.c_str();
}

mz_status mz_load_model(const mz_model_cfg* cfg, const void* blob, size_t nbytes, int32_t device,
                        mz_ctx** out) {
  if (out) *out = nullptr;
  std::unique_ptr<mz_ctx> x(new (std::nothrow) mz_ctx());
  if (!x) {
    g_load_error = "host allocation failed";
    return MZ_ENOMEM;
  }
  mz_ctx* raw = x.get();
  mz_status st = guarded(nullptr, [&] {
    if (!out) fail(MZ_EINVAL, "out is NULL");
    validate_cfg(cfg);
    if (!blob) fail(MZ_EINVAL, "blob is NULL");
    if ((int64_t)nbytes != blob_bytes(cfg))
      fail(MZ_EINVAL, "blob has %zu bytes, the configuration needs %lld", nbytes, (long long)blob_bytes(cfg));
    int ndev = 0;
    HIPCHK(hipGetDeviceCount(&ndev));
    if (device < 0 || device >= ndev) fail(MZ_EINVAL, "device %d not present (%d devices)", device, ndev);
    raw->device = device;
    HIPCHK(hipSetDevice(device));
    raw->cfg = *cfg;
    mz_ctx& c = *raw;
    c.L = cfg->n_layers; c.d = cfg->d_model; c.nq = cfg->n_q_heads; c.nkv = cfg->n_kv_heads;
    c.hd = cfg->head_dim; c.ff = cfg->d_ffn; c.V = cfg->vocab; c.C = cfg->chunk_tokens;
    c.max_ctx = cfg->max_ctx;
    c.dq = c.nq * c.hd; c.dkv = c.nkv * c.hd;
    c.dq_pad = (int)round_up(c.dq, mzk::kGemmTileN);
    c.kv_pad = (int)round_up(2 * c.dkv, mzk::kGemmTileN);
    c.d_pad = (int)round_up(c.d, mzk::kGemmTileN);
    if (c.d_pad != c.d) fail(MZ_EINVAL, "d_model must be a multiple of %d", mzk::kGemmTileN);
    c.ffp = (int)round_up(c.ff, mzk::kGemmTileN / 2);
    c.max_chunks = c.nchunks_of(c.max_ctx);
    c.slot_bytes = (int64_t)c.C * c.dkv * 2 * 2;

    // weight unit layout
    const UnitLayout ul = unit_layout(*cfg);
    c.off_q = ul.off_q;
    c.off_kv = ul.off_kv;
    c.off_o = ul.off_o;
    c.off_gu = ul.off_gu;
    c.off_dn = ul.off_dn;
    c.unit_bytes = ul.unit_bytes;

    HIPCHK(hipStreamCreateWithFlags(&c.s_compute, hipStreamNonBlocking));
    HIPCHK(hipStreamCreateWithFlags(&c.s_swap, hipStreamNonBlocking));
    c.ev_w.resize(c.L);
    c.ev_kv.resize(c.L);
    for (int l = 0; l < c.L; ++l) {
      HIPCHK(hipEventCreateWithFlags(&c.ev_w[l], hipEventDisableTiming));
      HIPCHK(hipEventCreateWithFlags(&c.ev_kv[l], hipEventDisableTiming));
    }
    HIPCHK(hipEventCreate(&c.ev_swap_start));
    HIPCHK(hipEventCreate(&c.ev_swap_end));

    // repack layer units into a pinned host image, then upload
    void* img = nullptr;
    if (hipHostMalloc(&img, (size_t)c.unit_bytes * c.L, hipHostMallocDefault) != hipSuccess || !img)
      fail(MZ_ENOMEM, "pinned host allocation for the weight image failed");
    c.w_image = (uint8_t*)img;
    const uint8_t* bp = (const uint8_t*)blob;
    const int64_t rb_d = q4_row_bytes(c.d);
    for (int l = 0; l < c.L; ++l) {
      uint8_t* u = c.w_image + (int64_t)l * c.unit_bytes;
      memset(u, 0, c.unit_bytes);
      const uint8_t* wq = bp;                                  // Wq, Wk, Wv are consecutive rows
      const uint8_t* wo = wq + (int64_t)(c.dq + 2 * c.dkv) * rb_d;
      const uint8_t* wg = wo + (int64_t)c.d * q4_row_bytes(c.dq);
      const uint8_t* wu = wg + (int64_t)c.ff * rb_d;
      const uint8_t* wd = wu + (int64_t)c.ff * rb_d;
      pack_plain(wq, c.dq, c.d, u + c.off_q);
      pack_plain(wq + (int64_t)c.dq * rb_d, 2 * c.dkv, c.d, u + c.off_kv);
      pack_plain(wo, c.d, c.dq, u + c.off_o);
      pack_gateup(wg, wu, c.ff, c.d, u + c.off_gu);
      pack_plain(wd, c.d, c.ff, u + c.off_dn);
      bp = wd + (int64_t)c.d * q4_row_bytes(c.ff);
    }
    c.w_slab = (uint8_t*)dmalloc((size_t)c.unit_bytes * c.L);
    c.w_pool.init(c.L);
    c.w_slot.resize(c.L);
    c.w_state.assign(c.L, MZ_RES);
    c.w_entry.resize(c.L);
    for (int l = 0; l < c.L; ++l) c.w_slot[l] = c.w_pool.alloc_one();
    HIPCHK(hipMemcpy(c.w_slab, c.w_image, (size_t)c.unit_bytes * c.L, hipMemcpyHostToDevice));

    // embedding and output head, split into nibble and scale planes
    {
      const int64_t nib_b = (int64_t)c.V * c.d / 2, sc_b = (int64_t)c.V * (c.d / 32) * 2;
      std::vector<uint8_t> nib(nib_b);
      std::vector<uint16_t> sc((size_t)c.V * (c.d / 32));
      c.emb_nib = (uint8_t*)dmalloc(nib_b);
      c.emb_sc = (uint16_t*)dmalloc(sc_b);
      c.lm_nib = (uint8_t*)dmalloc(nib_b);
      c.lm_sc = (uint16_t*)dmalloc(sc_b);
      split_rows(bp, c.V, c.d, nib.data(), sc.data());
      HIPCHK(hipMemcpy(c.emb_nib, nib.data(), nib_b, hipMemcpyHostToDevice));
      HIPCHK(hipMemcpy(c.emb_sc, sc.data(), sc_b, hipMemcpyHostToDevice));
      split_rows(bp + (int64_t)c.V * rb_d, c.V, c.d, nib.data(), sc.data());
      HIPCHK(hipMemcpy(c.lm_nib, nib.data(), nib_b, hipMemcpyHostToDevice));
      HIPCHK(hipMemcpy(c.lm_sc, sc.data(), sc_b, hipMemcpyHostToDevice));
    }
    // RoPE table: angles in double precision, stored as float (cos, sin)
    {
      const int half = c.hd / 2;
      std::vector<float2> cs((size_t)c.max_ctx * half);
      for (int p = 0; p < c.max_ctx; ++p)
        for (int i = 0; i < half; ++i) {
          const double inv = std::pow((double)cfg->rope_theta, -2.0 * i / c.hd);
          const double a = (double)p * inv;
          cs[(size_t)p * half + i] = make_float2((float)std::cos(a), (float)std::sin(a));
        }
      c.rope_cs = (float2*)dmalloc(cs.size() * sizeof(float2));
      HIPCHK(hipMemcpy(c.rope_cs, cs.data(), cs.size() * sizeof(float2), hipMemcpyHostToDevice));
    }
    // KV slab
    const int n_slots = c.L * c.max_chunks;
    c.kv_slab = (uint8_t*)dmalloc((size_t)n_slots * c.slot_bytes);
    HIPCHK(hipMemset(c.kv_slab, 0, (size_t)n_slots * c.slot_bytes));
    c.kv_pool.init(n_slots);
    c.table.assign((size_t)c.L * c.max_chunks, -1);
    c.kv_state.assign((size_t)c.L * c.max_chunks, MZ_RES);
    c.kv_entry.resize((size_t)c.L * c.max_chunks);

    // activations
    const int64_t M = c.max_ctx;
    c.h[0] = (float*)dmalloc((size_t)M * c.d * 4);
    c.h[1] = (float*)dmalloc((size_t)M * c.d * 4);
    c.xb = dmalloc((size_t)M * std::max(c.d, c.dq) * 2);
    c.qf = (float*)dmalloc((size_t)M * c.dq_pad * 4);
    c.kvf = (float*)dmalloc((size_t)M * c.kv_pad * 4);
    c.q16 = dmalloc((size_t)M * c.dq * 2);
    c.act = dmalloc((size_t)M * c.ffp * 2);
    c.logits = (float*)dmalloc((size_t)c.V * 4);
    const int nblk = (c.V + 63) / 64;
    c.part_val = (float*)dmalloc((size_t)nblk * 4);
    c.part_idx = (int32_t*)dmalloc((size_t)nblk * 4);
    c.d_token = (int32_t*)dmalloc(4);
    c.d_gen = (int32_t*)dmalloc((size_t)c.max_ctx * 4);

    // restore metadata
    const int64_t tot = (int64_t)c.L * M;
    // tables and compressed-chunk slots (4 + 4 bytes per layer and chunk),
    // five per-row arrays (24 bytes per layer and row), tokens, alignment
    c.stage_bytes = (size_t)c.L * c.max_chunks * 8 + (size_t)tot * 24 + (size_t)M * 4 + 9 * 256;
    c.d_meta = (uint8_t*)dmalloc(c.stage_bytes);
    c.comp_bytes = mzk::kv_compressed_bytes(c.slot_bytes / 2);
    c.split_ws_bytes = std::min<int64_t>(
        int64_t(64) << 20, std::max(mzk::attention_split_ws_bytes(std::min<int64_t>(M, 4096), c.nq, c.hd, 64),
                                    mzk::gemm_splitk_ws_bytes(std::min<int64_t>(M, 512), 2 * c.ffp, 8)));
    c.split_ws = (uint8_t*)dmalloc((size_t)c.split_ws_bytes);
    c.attn_wq = (int32_t*)dmalloc(mzk::kAttnQueueInts * sizeof(int32_t));
    HIPCHK(hipMemset(c.attn_wq, 0, mzk::kAttnQueueInts * sizeof(int32_t)));
    c.gemm_wq = (int32_t*)dmalloc(mzk::kGemmQueueInts * sizeof(int32_t));
    HIPCHK(hipMemset(c.gemm_wq, 0, mzk::kGemmQueueInts * sizeof(int32_t)));
    HIPCHK(hipEventCreateWithFlags(&c.ev_meta, hipEventDisableTiming));
    void* stage = nullptr;
    if (hipHostMalloc(&stage, c.stage_bytes, hipHostMallocDefault) != hipSuccess || !stage)
      fail(MZ_ENOMEM, "pinned staging allocation failed");
    c.h_stage = (uint8_t*)stage;
    void* tokp = nullptr;
    if (hipHostMalloc(&tokp, 64, hipHostMallocDefault) != hipSuccess || !tokp)
      fail(MZ_ENOMEM, "pinned allocation failed");
    c.h_token = (int32_t*)tokp;
    HIPCHK(hipDeviceSynchronize());
  });
  if (st != MZ_OK) {
    mz_free(x.release());
    return st;
  }
  *out = x.release();
  return MZ_OK;
}

void mz_free(mz_ctx* x) {
  if (!x) return;
  (void)hipSetDevice(x->device);
  if (x->s_compute) (void)hipStreamSynchronize(x->s_compute);
  if (x->s_swap) (void)hipStreamSynchronize(x->s_swap);
  void* dptrs[] = {x->codec_stage, x->d_meta, x->split_ws, x->attn_wq, x->gemm_wq, x->w_slab, x->emb_nib, x->emb_sc, x->lm_nib, x->lm_sc,
                   x->rope_cs, x->kv_slab,
                   x->h[0], x->h[1], x->xb, x->qf, x->kvf, x->q16, x->act, x->logits, x->part_val,
                   x->part_idx, x->d_token, x->d_gen};
  for (void* p : dptrs)
    if (p) (void)hipFree(p);
  if (x->w_image) (void)hipHostFree(x->w_image);
  if (x->h_stage) (void)hipHostFree(x->h_stage);
  if (x->h_token) (void)hipHostFree(x->h_token);
  x->arena.release_all();
  for (auto e : x->ev_w) if (e) (void)hipEventDestroy(e);
  for (auto e : x->ev_kv) if (e) (void)hipEventDestroy(e);
  for (auto e : x->ev_pool) (void)hipEventDestroy(e);
  if (x->ev_swap_start) (void)hipEventDestroy(x->ev_swap_start);
  if (x->ev_swap_end) (void)hipEventDestroy(x->ev_swap_end);
  if (x->ev_meta) (void)hipEventDestroy(x->ev_meta);
  if (x->s_compute) (void)hipStreamDestroy(x->s_compute);
  if (x->s_swap) (void)hipStreamDestroy(x->s_swap);
  delete x;
}

mz_status mz_set_option(mz_ctx* x, const char* key, int64_t value) {
  if (!x) return MZ_EINVAL;
  return guarded(x, [&] {
    if (!key) fail(MZ_EINVAL, "key is NULL");
    const std::string k(key);
    if (k == "overlap") x->overlap = value != 0;
    else if (k == "debug_swap_delay_us") x->debug_swap_delay_us = value < 0 ? 0 : value;
    else if (k == "debug_poison") x->debug_poison = value != 0;
    else if (k == "debug_kv_slot_limit") x->kv_pool.limit = value < 0 ? -1 : (int)std::min<int64_t>(value, INT32_MAX);
    else if (k == "swap_trim") x->swap_trim = value != 0;
    else if (k == "attn_split") x->attn_split = value != 0;
    else if (k == "attn_queue") x->attn_queue = value != 0;
    else if (k == "gemm_queue") x->gemm_queue = value != 0;
    else if (k == "gemm_split") x->gemm_split = value != 0;
    else if (k == "gemv_direct") x->gemv_direct = value != 0;
    else if (k == "gemv_qkv") x->gemv_qkv = value != 0;
    else if (k == "fuse_norm") x->fuse_norm = value != 0;
    else if (k == "fuse_rope") x->fuse_rope = value != 0;
    else if (k == "kv_codec") {
      if (value && !x->codec_stage) {
        HIPCHK(hipMalloc((void**)&x->codec_stage, (size_t)x->max_chunks * (size_t)x->comp_bytes));
      }
      x->kv_codec = value != 0;
    }
    else if (k == "kernel_timing") {
      HIPCHK(hipStreamSynchronize(x->s_compute));
      x->collect_timing();
      x->timing = value != 0;
      for (auto& s : x->kstats) s = KindStats();
    } else fail(MZ_EINVAL, "unknown option '%s'", key);
  });
}

static void check_tokens(const mz_ctx* x, const int32_t* t, int32_t n) {
  if (n < 0) fail(MZ_EINVAL, "token count is negative");
  if (n > 0 && !t) fail(MZ_EINVAL, "tokens is NULL");
  if (n > x->max_ctx) fail(MZ_EINVAL, "%d tokens exceed max_ctx (%d)", n, x->max_ctx);
  for (int i = 0; i < n; ++i)
    if (t[i] < 0 || t[i] >= x->V) fail(MZ_EINVAL, "token %d out of range", t[i]);
}

mz_status mz_prefill_context(mz_ctx* x, const int32_t* tokens, int32_t n) {
  if (!x) return MZ_EINVAL;
  return guarded(x, [&] {
    check_tokens(x, tokens, n);
    if (n == 0) fail(MZ_EINVAL, "empty context");
    HIPCHK(hipStreamSynchronize(x->s_compute));
    HIPCHK(hipStreamSynchronize(x->s_swap));
    // weights must be resident for a clean prefill: bring evicted units back
    x->release_context();
    restore_and_prefill_impl(x, tokens, n);
  });
}

mz_status mz_set_context(mz_ctx* x, const int32_t* tokens, int32_t n) {
  if (!x) return MZ_EINVAL;
  return guarded(x, [&] {
    check_tokens(x, tokens, n);
    HIPCHK(hipStreamSynchronize(x->s_compute));
    HIPCHK(hipStreamSynchronize(x->s_swap));
    x->release_context();
    const int nc = x->nchunks_of(n);
    for (int l = 0; l < x->L; ++l)
      for (int c = 0; c < nc; ++c) {
        int s = x->kv_pool.alloc_one();
        if (s < 0) fail(MZ_ENOMEM, "KV slot pool exhausted");
        x->table[(size_t)l * x->max_chunks + c] = s;
        mzk::launch_zero(x->kv_slab + (int64_t)s * x->slot_bytes, x->slot_bytes / 4, x->s_compute);
      }
    HIPCHK(hipGetLastError());
    HIPCHK(hipStreamSynchronize(x->s_compute));
    x->tokens.assign(tokens, tokens + n);
  });
}

mz_status mz_truncate_context(mz_ctx* x, int32_t n) {
  if (!x) return MZ_EINVAL;
  return guarded(x, [&] {
    if (n < 0 || n > (int)x->tokens.size()) fail(MZ_EINVAL, "n=%d outside 0..%zu", n, x->tokens.size());
    const int nc = x->nchunks_of((int)x->tokens.size()), keep = x->nchunks_of(n);
    for (int l = 0; l < x->L; ++l) {
      if (x->w_state[l] != MZ_RES) fail(MZ_ESTATE, "weights of layer %d are evicted", l);
      for (int c = 0; c < nc; ++c)
        if (x->kv_state[(size_t)l * x->max_chunks + c] != MZ_RES) fail(MZ_ESTATE, "KV chunks are evicted");
    }
    HIPCHK(hipStreamSynchronize(x->s_compute));
    HIPCHK(hipStreamSynchronize(x->s_swap));
    for (int l = 0; l < x->L; ++l)
      for (int c = keep; c < nc; ++c) {
        int32_t& t = x->table[(size_t)l * x->max_chunks + c];
        if (t >= 0) x->kv_pool.release(t);
        t = -1;
      }
    x->tokens.resize(n);
    x->have_last = false;
  });
}

static int32_t chunk_slot(mz_ctx* x, int32_t layer, int32_t chunk) {
  if (layer < 0 || layer >= x->L) fail(MZ_EINVAL, "layer %d out of range", layer);
  const int nc = x->nchunks_of((int)x->tokens.size());
  if (chunk < 0 || chunk >= nc) fail(MZ_EINVAL, "chunk %d out of range (%d chunks)", chunk, nc);
  const int32_t s = x->table[(size_t)layer * x->max_chunks + chunk];
  if (s < 0 || x->kv_state[(size_t)layer * x->max_chunks + chunk] != MZ_RES)
    fail(MZ_ESTATE, "chunk (%d, %d) is not resident", layer, chunk);
  return s;
}

// The exchange layout of a chunk is K [C][dkv] and V [C][dkv]; the slot keeps
// V dimension-major (V^T [dkv][C]) for the attention kernel, so V is
// transposed on the way in and out.
static void transpose_f16(const uint16_t* in, int rows, int cols, uint16_t* out) {
  for (int r = 0; r < rows; ++r)
    for (int c = 0; c < cols; ++c) out[(size_t)c * rows + r] = in[(size_t)r * cols + c];
}

mz_status mz_import_kv(mz_ctx* x, int32_t layer, int32_t chunk, const void* k, const void* v) {
  if (!x) return MZ_EINVAL;
  return guarded(x, [&] {
    if (!k || !v) fail(MZ_EINVAL, "k or v is NULL");
    const int32_t s = chunk_slot(x, layer, chunk);
    HIPCHK(hipStreamSynchronize(x->s_compute));
    const size_t half = (size_t)x->slot_bytes / 2;
    std::vector<uint16_t> vt((size_t)x->C * x->dkv);
    transpose_f16((const uint16_t*)v, x->C, x->dkv, vt.data());
    uint8_t* dst = x->kv_slab + (int64_t)s * x->slot_bytes;
    HIPCHK(hipMemcpy(dst, k, half, hipMemcpyHostToDevice));
    HIPCHK(hipMemcpy(dst + half, vt.data(), half, hipMemcpyHostToDevice));
  });
}

mz_status mz_read_kv(mz_ctx* x, int32_t layer, int32_t chunk, void* k, void* v) {
  if (!x) return MZ_EINVAL;
  return guarded(x, [&] {
    if (!k || !v) fail(MZ_EINVAL, "k or v is NULL");
    const int32_t s = chunk_slot(x, layer, chunk);
    HIPCHK(hipStreamSynchronize(x->s_compute));
    HIPCHK(hipStreamSynchronize(x->s_swap));
    const size_t half = (size_t)x->slot_bytes / 2;
    std::vector<uint16_t> vt((size_t)x->C * x->dkv);
    const uint8_t* src = x->kv_slab + (int64_t)s * x->slot_bytes;
    HIPCHK(hipMemcpy(k, src, half, hipMemcpyDeviceToHost));
    HIPCHK(hipMemcpy(vt.data(), src + half, half, hipMemcpyDeviceToHost));
    transpose_f16(vt.data(), x->dkv, x->C, (uint16_t*)v);
  });
}

mz_status mz_evict(mz_ctx* x, const mz_evict_plan* plan) {
  if (!x) return MZ_EINVAL;
  return guarded(x, [&] {
    if (!plan || !plan->kv_state) fail(MZ_EINVAL, "plan or plan->kv_state is NULL");
    const int L = x->L, MC = x->max_chunks;
    const int nc = x->nchunks_of((int)x->tokens.size());
    if (x->tokens.empty()) fail(MZ_ESTATE, "no cached context to evict");
    if (plan->n_layers != L || plan->n_chunks != nc)
      fail(MZ_EINVAL, "plan is %dx%d, the context has %dx%d units", plan->n_layers, plan->n_chunks, L, nc);
    const int n_units = L * nc + L;
    auto target = [&](int u) -> int {
      return u < L * nc ? plan->kv_state[u] : (plan->w_state ? plan->w_state[u - L * nc] : MZ_RES);
    };
    auto current = [&](int u) -> int {
      return u < L * nc ? x->kv_state[(size_t)(u / nc) * MC + u % nc] : x->w_state[u - L * nc];
    };
    // visiting order: the given order, then every other unit backward-out
    std::vector<int> order;
    std::vector<char> seen(n_units, 0);
    if (plan->order) {
      if (plan->n_order < 0) fail(MZ_EINVAL, "n_order is negative");
      for (int i = 0; i < plan->n_order; ++i) {
        const int u = plan->order[i];
        if (u < 0 || u >= n_units || seen[u]) fail(MZ_EINVAL, "order entry %d invalid or repeated", u);
        seen[u] = 1;
        order.push_back(u);
      }
    }
    for (int l = L - 1; l >= 0; --l) {
      for (int c = nc - 1; c >= 0; --c)
        if (!seen[l * nc + c]) order.push_back(l * nc + c);
      if (!seen[L * nc + l]) order.push_back(L * nc + l);
    }
    // validate before touching anything
    for (int u = 0; u < n_units; ++u) {
      const int t = target(u), cur = current(u);
      if (t != MZ_RES && t != MZ_SWAP && t != MZ_DROP) fail(MZ_EINVAL, "unit %d: state %d invalid", u, t);
      if (t == MZ_SWAP && cur == MZ_DROP) fail(MZ_ESTATE, "unit %d is dropped and cannot be swapped", u);
    }
    HIPCHK(hipStreamSynchronize(x->s_compute));
    HIPCHK(hipStreamSynchronize(x->s_swap));
    x->collect_timing();
    std::vector<int> release_kv;
    std::vector<int> release_w;
    int64_t n_comp = 0;
    for (int u : order) {
      const int t = target(u), cur = current(u);
      if (t == MZ_RES || t == cur) continue;
      if (u < L * nc) {
        const int l = u / nc, c = u % nc;
        const size_t idx = (size_t)l * MC + c;
        if (t == MZ_SWAP) {
          const uint8_t* slot = x->kv_slab + (int64_t)x->table[idx] * x->slot_bytes;
          const bool full = (int64_t)(c + 1) * x->C <= (int64_t)x->tokens.size();
          if (x->kv_codec && full) {
            // compress into the staging ring, then copy the compressed bytes out
            uint8_t* stage = x->codec_stage + (n_comp++ % x->max_chunks) * x->comp_bytes;
            mzk::launch_kv_compress(slot, nullptr, 0, x->slot_bytes / 2, 1, stage, x->s_swap);
            HIPCHK(hipGetLastError());
            const ArenaEntry e = x->arena.push((size_t)x->comp_bytes);
            HIPCHK(hipMemcpyAsync(x->arena.ptr(e), stage, x->comp_bytes, hipMemcpyDeviceToHost, x->s_swap));
            x->kv_entry[idx] = e;
          } else {
            const ArenaEntry e = x->arena.push((size_t)x->slot_bytes);
            HIPCHK(hipMemcpyAsync(x->arena.ptr(e), slot, x->slot_bytes, hipMemcpyDeviceToHost, x->s_swap));
            x->kv_entry[idx] = e;
          }
        }
        if (cur == MZ_RES) release_kv.push_back(x->table[idx]);
        x->table[idx] = -1;
        x->kv_state[idx] = (uint8_t)t;
      } else {
        const int l = u - L * nc;
        if (t == MZ_SWAP) {
          const ArenaEntry e = x->arena.push((size_t)x->unit_bytes);
          HIPCHK(hipMemcpyAsync(x->arena.ptr(e), x->unit_ptr(l), x->unit_bytes, hipMemcpyDeviceToHost,
                                x->s_swap));
          x->w_entry[l] = e;
        }
        if (cur == MZ_RES) release_w.push_back(x->w_slot[l]);
        x->w_slot[l] = -1;
        x->w_state[l] = (uint8_t)t;
      }
    }
    HIPCHK(hipStreamSynchronize(x->s_swap));
    for (int s : release_kv) x->kv_pool.release(s);
    for (int s : release_w) x->w_pool.release(s);
    x->have_last = false;
  });
}

mz_status mz_evict_size(mz_ctx* x, const mz_evict_size_request* req, double* info) {
  if (!x) return MZ_EINVAL;
  std::vector<uint8_t> kv, ws;
  std::vector<int32_t> order;
  int32_t n_ev = 0;
  int32_t L = 0, nc = 0;
  mz_status st = guarded(x, [&] {
    if (!req) fail(MZ_EINVAL, "req is NULL");
    if (x->tokens.empty()) fail(MZ_ESTATE, "no cached context to evict");
    L = x->L;
    nc = x->nchunks_of((int)x->tokens.size());
    kv.resize((size_t)L * nc);
    for (int l = 0; l < L; ++l)
      for (int c = 0; c < nc; ++c) kv[(size_t)l * nc + c] = x->kv_state[(size_t)l * x->max_chunks + c];
    ws.assign(x->w_state.begin(), x->w_state.end());
    order.resize((size_t)L * (nc + 1));
    mz_evict_size_request r = *req;
    r.kv_codec = x->kv_codec ? 1 : 0;
    if (mz_plan_evict_size(&x->cfg, (int32_t)x->tokens.size(), &r, kv.data(), ws.data(), order.data(), nullptr,
                           &n_ev, info) != MZ_OK)
      fail(MZ_EINVAL, "%s", mz_last_error(nullptr));
  });
  if (st != MZ_OK || n_ev == 0) return st;
  mz_evict_plan plan{};
  plan.n_layers = L;
  plan.n_chunks = nc;
  plan.kv_state = kv.data();
  plan.w_state = ws.data();
  plan.order = order.data();
  plan.n_order = n_ev;
  return mz_evict(x, &plan);
}

mz_status mz_restore_and_prefill(mz_ctx* x, const int32_t* prompt, int32_t n_prompt) {
  if (!x) return MZ_EINVAL;
  return guarded(x, [&] {
    if (x->tokens.empty() && n_prompt == 0) fail(MZ_ESTATE, "no cached context and no prompt");
    if (n_prompt > 0) check_tokens(x, prompt, n_prompt);
    restore_and_prefill_impl(x, prompt, n_prompt);
  });
}

mz_status mz_first_token(mz_ctx* x, int32_t* token_out, float* logits_out) {
  if (!x) return MZ_EINVAL;
  return guarded(x, [&] {
    if (!token_out) fail(MZ_EINVAL, "token_out is NULL");
    if (!x->have_last) fail(MZ_ESTATE, "no prefill since the last first token");
    hipStream_t cs = x->s_compute;
    x->timed(kKLmHead, 2.0 * x->d * x->V, (double)x->V * x->d * 0.5625 + x->V * 4.0, cs, [&] {
      mzk::launch_lm_head(x->h_last, x->d, x->cfg.rms_eps, x->lm_nib, x->lm_sc, x->V, x->logits,
                          x->part_val, x->part_idx, x->d_token, cs);
    });
    HIPCHK(hipMemcpyAsync(x->h_token, x->d_token, 4, hipMemcpyDeviceToHost, cs));
    if (logits_out)
      HIPCHK(hipMemcpyAsync(logits_out, x->logits, (size_t)x->V * 4, hipMemcpyDeviceToHost, cs));
    HIPCHK(hipStreamSynchronize(cs));
    *token_out = *x->h_token;
    x->have_last = false;
    if (x->swap_timed) {
      HIPCHK(hipEventSynchronize(x->ev_swap_end));
      float ms = 0;
      HIPCHK(hipEventElapsedTime(&ms, x->ev_swap_start, x->ev_swap_end));
      x->last_swap_ms = ms;
      x->swap_timed = false;
    }
    x->collect_timing();
  });
}

mz_status mz_generate(mz_ctx* x, int32_t token, int32_t n, int32_t* tokens_out) {
  if (!x) return MZ_EINVAL;
  if (n < 0 || (n > 0 && !tokens_out)) return guarded(x, [&] { fail(MZ_EINVAL, "bad n or tokens_out"); });
  if (n == 0) return MZ_OK;
  // the first step as a restore and first token of its own (it may bring
  // back evicted units and time their copies)
  mz_status st = mz_restore_and_prefill(x, &token, 1);
  if (st != MZ_OK) return st;
  st = mz_first_token(x, &tokens_out[0], nullptr);
  if (st != MZ_OK || n == 1) return st;
  // the others back to back: each step's token stays on the device, where
  // the argmax leaves it (d_gen[i]) and the next step's embedding reads it;
  // the host plans the next step while the GPU runs this one and learns
  // the tokens at the end (the context records placeholders until then)
  return guarded(x, [&] {
    const size_t base = x->tokens.size();   // position at which step 1 prefills tokens_out[0]
    if ((int64_t)n > (int64_t)x->max_ctx) fail(MZ_EINVAL, "n exceeds max_ctx");
    hipStream_t cs = x->s_compute;
    int done = 1;   // steps 0 .. done - 1 are enqueued (and their tokens final after settle)
    auto settle = [&]() {
      HIPCHK(hipStreamSynchronize(cs));
      if (done > 1)
        HIPCHK(hipMemcpy(&tokens_out[1], x->d_gen + 1, (size_t)(done - 1) * 4, hipMemcpyDeviceToHost));
      // step i >= 2 prefilled tokens_out[i - 1] at position base + i - 1
      for (int i = 2; i < done; ++i) x->tokens[base + i - 1] = tokens_out[i - 1];
    };
    try {
      for (int i = 1; i < n; ++i) {
        const int32_t placeholder = 0;
        if (i == 1)
          restore_and_prefill_impl(x, &tokens_out[0], 1);
        else
          restore_and_prefill_impl(x, &placeholder, 1, x->d_gen + (i - 1));
        x->timed(kKLmHead, 2.0 * x->d * x->V, (double)x->V * x->d * 0.5625 + x->V * 4.0, cs, [&] {
          mzk::launch_lm_head(x->h_last, x->d, x->cfg.rms_eps, x->lm_nib, x->lm_sc, x->V, x->logits,
                              x->part_val, x->part_idx, x->d_token, cs, x->d_gen + i);
        });
        x->have_last = false;
        done = i + 1;
      }
    } catch (...) {
      try {
        settle();
      } catch (...) {
      }
      throw;
    }
    settle();
  });
}

mz_status mz_stats(mz_ctx* x, char* out, size_t cap) {
  if (!x) return MZ_EINVAL;
  return guarded(x, [&] {
    if (!out) fail(MZ_EINVAL, "json_out is NULL");
    std::string s = "{";
    char buf[512];
    snprintf(buf, sizeof buf, "\"version\": \"%s\", \"n_ctx\": %zu, \"last_N\": %d, \"last_P\": %d, ",
             kVersion, x->tokens.size(), x->last_N, x->last_P);
    s += buf;
    auto arr = [&](const char* name, const std::vector<int32_t>& v) {
      s += "\""; s += name; s += "\": [";
      for (size_t i = 0; i < v.size(); ++i) {
        if (i) s += ", ";
        s += std::to_string(v[i]);
      }
      s += "], ";
    };
    arr("nR", x->last_nR);
    arr("nD", x->last_nD);
    arr("nQ", x->last_nQ);
    snprintf(buf, sizeof buf,
             "\"swap_kv_bytes\": %lld, \"swap_w_bytes\": %lld, \"reload_w_bytes\": %lld, \"copies\": %lld, "
             "\"swap_ms\": %.6f, \"algo_flops\": %.6e, \"host_plan_ms\": %.4f, \"host_enqueue_ms\": %.4f, ",
             (long long)x->last_swap_kv_bytes, (long long)x->last_swap_w_bytes,
             (long long)x->last_reload_w_bytes, (long long)x->last_copies, x->last_swap_ms,
             x->last_algo_flops, x->last_plan_ms, x->last_enqueue_ms);
    s += buf;
    snprintf(buf, sizeof buf,
             "\"pool\": {\"kv_slots\": %d, \"kv_slots_used\": %d, \"slot_bytes\": %lld, \"w_units\": %d, "
             "\"w_units_used\": %d, \"unit_bytes\": %lld, \"arena_reserved\": %zu}, ",
             x->kv_pool.n, x->kv_pool.used(), (long long)x->slot_bytes, x->w_pool.n, x->w_pool.used(),
             (long long)x->unit_bytes, x->arena.reserved());
    s += buf;
    s += "\"kernels\": {";
    bool first = true;
    for (int k = 0; k < kKCount; ++k) {
      const KindStats& ks = x->kstats[k];
      if (!ks.launches) continue;
      snprintf(buf, sizeof buf,
               "%s\"%s\": {\"kernel\": \"%s\", \"launches\": %lld, \"ms\": %.6f, \"flops\": %.6e, \"bytes\": %.6e}",
               first ? "" : ", ", kKindName[k], kKindKernel[k], (long long)ks.launches, ks.ms, ks.flops,
               ks.bytes);
      s += buf;
      first = false;
    }
    s += "}}";
    if (s.size() + 1 > cap) fail(MZ_EINVAL, "json buffer needs %zu bytes", s.size() + 1);
    memcpy(out, s.c_str(), s.size() + 1);
  });
}

mz_status mz_plan_rows(const mz_model_cfg* cfg, const uint8_t* kv_state, int32_t n_chunks, int32_t n_ctx,
                       int32_t n_prompt, int32_t* nR, int32_t* nD, int32_t* rows_out, int64_t rows_cap) {
  return guarded(nullptr, [&] {
    if (!cfg || !kv_state || !nR || !nD) fail(MZ_EINVAL, "NULL argument");
    if (cfg->n_layers < 1 || cfg->chunk_tokens < 1) fail(MZ_EINVAL, "bad cfg");
    if (n_ctx < 0 || n_prompt < 0 || n_ctx + n_prompt < 1) fail(MZ_EINVAL, "bad token counts");
    if (n_chunks != (n_ctx + cfg->chunk_tokens - 1) / cfg->chunk_tokens) fail(MZ_EINVAL, "n_chunks mismatch");
    for (int64_t i = 0; i < (int64_t)cfg->n_layers * n_chunks; ++i)
      if (kv_state[i] > MZ_DROP) fail(MZ_EINVAL, "bad state value");
    Rows r = compute_rows(kv_state, cfg->n_layers, n_chunks, n_ctx, n_prompt, cfg->chunk_tokens);
    int64_t tot = 0;
    for (int l = 0; l < cfg->n_layers; ++l) {
      nR[l] = r.nR[l];
      nD[l] = r.nD[l];
      tot += r.nR[l];
    }
    if (rows_out) {
      if (tot > rows_cap) fail(MZ_EINVAL, "rows_cap %lld < %lld", (long long)rows_cap, (long long)tot);
      int64_t o = 0;
      for (auto& v : r.R)
        for (int32_t p : v) rows_out[o++] = p;
    }
  });
}

int64_t mz_q4_gemm_packed_bytes(int32_t n, int32_t k) {
  if (n < 1 || k < 1) return 0;
  return gemm_packed_bytes(n, k);
}

mz_status mz_q4_gemm_pack(const void* w, const void* w_up, int32_t n, int32_t k, void* out) {
  return guarded(nullptr, [&] {
    if (!w || !out || n < 1 || k < 1) fail(MZ_EINVAL, "bad arguments");
    if (w_up)
      pack_gateup((const uint8_t*)w, (const uint8_t*)w_up, n, k, (uint8_t*)out);
    else
      pack_plain((const uint8_t*)w, n, k, (uint8_t*)out);
  });
}

static mz_status gemm_entry(const void* x_f16, int32_t m, int32_t n_pad, int32_t k, const void* w_packed,
                            int32_t epilogue, void* y, int32_t* queues, void* stream) {
  return guarded(nullptr, [&] {
    if (!x_f16 || !w_packed || !y) fail(MZ_EINVAL, "NULL pointer");
    if (m < 1 || n_pad < 1 || k < 1) fail(MZ_EINVAL, "sizes must be positive");
    if (n_pad % mzk::kGemmTileN) fail(MZ_EINVAL, "n_pad must be a multiple of %d", mzk::kGemmTileN);
    if (k % mzk::kGemmTileK) fail(MZ_EINVAL, "k must be a multiple of %d", mzk::kGemmTileK);
    if (epilogue < 0 || epilogue > 2) fail(MZ_EINVAL, "bad epilogue");
    mzk::launch_gemm_q4(x_f16, m, n_pad, k, w_packed, epilogue, y, (hipStream_t)stream, nullptr, queues);
    HIPCHK(hipGetLastError());
  });
}

mz_status mz_q4_gemm(const void* x_f16, int32_t m, int32_t n_pad, int32_t k, const void* w_packed,
                     int32_t epilogue, void* y, void* stream) {
  return gemm_entry(x_f16, m, n_pad, k, w_packed, epilogue, y, nullptr, stream);
}

mz_status mz_q4_gemm_queued(const void* x_f16, int32_t m, int32_t n_pad, int32_t k, const void* w_packed,
                            int32_t epilogue, void* y, int32_t* work_queues, void* stream) {
  if (!work_queues) return guarded(nullptr, [&] { fail(MZ_EINVAL, "work_queues is NULL"); });
  return gemm_entry(x_f16, m, n_pad, k, w_packed, epilogue, y, work_queues, stream);
}

mz_status mz_q4_gemm_ex(const void* x_f16, int32_t m, int32_t n_pad, int32_t k, const void* w_packed,
                        int32_t epilogue, const mz_q4_gemm_args* args, void* y, void* stream) {
  return guarded(nullptr, [&] {
    const mz_q4_gemm_args a = args ? *args : mz_q4_gemm_args{};
    if (!x_f16 || !w_packed) fail(MZ_EINVAL, "NULL pointer");
    if (m < 1 || n_pad < 1 || k < 1) fail(MZ_EINVAL, "sizes must be positive");
    if (n_pad % mzk::kGemmTileN) fail(MZ_EINVAL, "n_pad must be a multiple of %d", mzk::kGemmTileN);
    if (k % mzk::kGemmTileK) fail(MZ_EINVAL, "k must be a multiple of %d", mzk::kGemmTileK);
    if (a.workspace_bytes < 0 || (a.workspace_bytes > 0 && !a.workspace)) fail(MZ_EINVAL, "bad workspace");
    hipStream_t s = (hipStream_t)stream;
    if (epilogue >= 0 && epilogue <= 2) {
      if (!y) fail(MZ_EINVAL, "NULL y");
      mzk::launch_gemm_q4(x_f16, m, n_pad, k, w_packed, epilogue, y, s, a.a_rows, a.work_queues, a.workspace,
                          a.workspace_bytes);
    } else if (epilogue == mzk::kEpiRopeQ || epilogue == mzk::kEpiRopeKV) {
      if (!a.pos || !a.rope_cs) fail(MZ_EINVAL, "the rotary epilogues need pos and rope_cs");
      if (epilogue == mzk::kEpiRopeQ && !y) fail(MZ_EINVAL, "NULL y");
      if (epilogue == mzk::kEpiRopeKV && (!a.kv_off || !a.slab)) fail(MZ_EINVAL, "epilogue 5 needs kv_off and slab");
      if (!mzk::gemm_rope_fusable(a.head_dim, epilogue == mzk::kEpiRopeKV ? a.chunk_tokens : 1))
        fail(MZ_EINVAL, "head_dim must be 32, 64 or 128 and chunk_tokens a power of two");
      if (a.n_valid < 1 || a.n_valid > n_pad || a.n_valid % (epilogue == mzk::kEpiRopeKV ? 2 * a.head_dim : a.head_dim))
        fail(MZ_EINVAL, "n_valid must be whole heads within n_pad");
      mzk::GemmRope ea;
      ea.pos = a.pos;
      ea.kv_off = a.kv_off;
      ea.rope_cs = reinterpret_cast<const float2*>(a.rope_cs);
      ea.slab = reinterpret_cast<uint8_t*>(a.slab);
      ea.hd = a.head_dim;
      ea.n_valid = a.n_valid;
      ea.C = epilogue == mzk::kEpiRopeKV ? a.chunk_tokens : 1;
      mzk::launch_gemm_q4_rope(x_f16, m, n_pad, k, w_packed, epilogue, ea, y, s, a.a_rows, nullptr, a.workspace,
                               a.workspace_bytes);
    } else {
      fail(MZ_EINVAL, "bad epilogue");
    }
    HIPCHK(hipGetLastError());
  });
}

mz_status mz_q4_gemv(const void* x_f16, int32_t k, const void* w_packed, int32_t n_pad, int32_t epilogue,
                     const mz_q4_gemm_args* args, const float* h_norm, float eps, void* y, void* stream) {
  return guarded(nullptr, [&] {
    const mz_q4_gemm_args a = args ? *args : mz_q4_gemm_args{};
    if ((!x_f16 && !h_norm) || !w_packed) fail(MZ_EINVAL, "NULL pointer");
    if (!mzk::gemv1_ok(n_pad, k))
      fail(MZ_EINVAL, "n_pad must be a positive multiple of %d and k of %d, k at most %d", mzk::kGemmTileN,
           mzk::kGemmTileK, mzk::kGemv1MaxK);
    if (h_norm && !(eps >= 0.f)) fail(MZ_EINVAL, "eps must be >= 0");
    if (a.work_queues || a.workspace) fail(MZ_EINVAL, "the single-row product takes no work queues or workspace");
    mzk::GemmRope ea;
    if (epilogue >= 0 && epilogue <= 2) {
      if (!y) fail(MZ_EINVAL, "NULL y");
    } else if (epilogue == mzk::kEpiRopeQ || epilogue == mzk::kEpiRopeKV) {
      if (!a.pos || !a.rope_cs) fail(MZ_EINVAL, "the rotary epilogues need pos and rope_cs");
      if (epilogue == mzk::kEpiRopeQ && !y) fail(MZ_EINVAL, "NULL y");
      if (epilogue == mzk::kEpiRopeKV && (!a.kv_off || !a.slab)) fail(MZ_EINVAL, "epilogue 5 needs kv_off and slab");
      if (!mzk::gemm_rope_fusable(a.head_dim, epilogue == mzk::kEpiRopeKV ? a.chunk_tokens : 1))
        fail(MZ_EINVAL, "head_dim must be 32, 64 or 128 and chunk_tokens a power of two");
      if (a.n_valid < 1 || a.n_valid > n_pad || a.n_valid % (epilogue == mzk::kEpiRopeKV ? 2 * a.head_dim : a.head_dim))
        fail(MZ_EINVAL, "n_valid must be whole heads within n_pad");
      ea.pos = a.pos;
      ea.kv_off = a.kv_off;
      ea.rope_cs = reinterpret_cast<const float2*>(a.rope_cs);
      ea.slab = reinterpret_cast<uint8_t*>(a.slab);
      ea.hd = a.head_dim;
      ea.n_valid = a.n_valid;
      ea.C = epilogue == mzk::kEpiRopeKV ? a.chunk_tokens : 1;
    } else {
      fail(MZ_EINVAL, "bad epilogue");
    }
    mzk::launch_gemv1(x_f16, n_pad, k, w_packed, epilogue, ea, y, (hipStream_t)stream, a.a_rows, h_norm, eps);
    HIPCHK(hipGetLastError());
  });
}

int64_t mz_q4_gemm_split_workspace_bytes(int32_t m, int32_t n_pad, int32_t n_split) {
  if (m < 1 || n_pad < 1 || n_split < 1) return -1;
  return mzk::gemm_splitk_ws_bytes(m, n_pad, n_split);
}

int32_t mz_q4_gemm_auto_splits(int32_t m, int32_t n_pad, int32_t k, int64_t workspace_bytes) {
  if (m < 1 || n_pad < mzk::kGemmTileN || k < mzk::kGemmTileK) return 1;
  return mzk::gemm_auto_splits(m, n_pad, k, workspace_bytes);
}

int32_t mz_q4_gemm_long_k_splits(int32_t m, int32_t n_pad, int32_t k, int64_t workspace_bytes) {
  if (m < 1 || n_pad < mzk::kGemmTileN || k < mzk::kGemmTileK) return 1;
  return mzk::gemm_long_k_splits(m, n_pad, k, workspace_bytes);
}

mz_status mz_q4_gemm_split(const void* x_f16, int32_t m, int32_t n_pad, int32_t k, const void* w_packed,
                           int32_t epilogue, void* y, int32_t n_split, void* workspace, int64_t workspace_bytes,
                           void* stream) {
  return guarded(nullptr, [&] {
    if (!x_f16 || !w_packed || !y || !workspace) fail(MZ_EINVAL, "NULL pointer");
    if (m < 1 || n_pad < 1 || k < 1) fail(MZ_EINVAL, "sizes must be positive");
    if (n_pad % mzk::kGemmTileN) fail(MZ_EINVAL, "n_pad must be a multiple of %d", mzk::kGemmTileN);
    if (k % mzk::kGemmTileK) fail(MZ_EINVAL, "k must be a multiple of %d", mzk::kGemmTileK);
    if (epilogue < 0 || epilogue > 2) fail(MZ_EINVAL, "bad epilogue");
    if (n_split < 1 || n_split > 1024) fail(MZ_EINVAL, "n_split must be 1..1024");
    if (workspace_bytes < mzk::gemm_splitk_ws_bytes(m, n_pad, n_split))
      fail(MZ_EINVAL, "workspace too small for %d splits", n_split);
    mzk::launch_gemm_q4_splitk(x_f16, m, n_pad, k, w_packed, epilogue, y, n_split, workspace,
                               (hipStream_t)stream);
    HIPCHK(hipGetLastError());
  });
}

static mz_status attention_entry(const void* q, const int32_t* qpos, int32_t m, const void* slab,
                                 const int32_t* table, int32_t n_table, int32_t chunk_tokens, int32_t n_q,
                                 int32_t n_kv, int32_t head_dim, void* out, int32_t* queues, void* stream) {
  return guarded(nullptr, [&] {
    if (!q || !qpos || !slab || !table || !out) fail(MZ_EINVAL, "NULL pointer");
    if (m < 1 || n_table < 1) fail(MZ_EINVAL, "sizes must be positive");
    if (n_table > mzk::kAttnTableMax) fail(MZ_EINVAL, "n_table above %d", mzk::kAttnTableMax);
    if (chunk_tokens < 8 || (chunk_tokens & (chunk_tokens - 1))) fail(MZ_EINVAL, "chunk_tokens must be a power of two >= 8");
    if (head_dim != 64 && head_dim != 128) fail(MZ_EINVAL, "head_dim must be 64 or 128");
    if (n_kv < 1 || n_q % n_kv || n_q / n_kv > 8) fail(MZ_EINVAL, "bad head counts");
    const int64_t slot_bytes = (int64_t)chunk_tokens * n_kv * head_dim * 2 * 2;
    mzk::launch_attention(q, qpos, m, slab, table, n_table, chunk_tokens, slot_bytes, n_q, n_kv, head_dim, out,
                          (hipStream_t)stream, queues);
    HIPCHK(hipGetLastError());
  });
}

mz_status mz_attention(const void* q, const int32_t* qpos, int32_t m, const void* slab, const int32_t* table,
                       int32_t n_table, int32_t chunk_tokens, int32_t n_q, int32_t n_kv, int32_t head_dim,
                       void* out, void* stream) {
  return attention_entry(q, qpos, m, slab, table, n_table, chunk_tokens, n_q, n_kv, head_dim, out, nullptr,
                         stream);
}

mz_status mz_attention_queued(const void* q, const int32_t* qpos, int32_t m, const void* slab,
                              const int32_t* table, int32_t n_table, int32_t chunk_tokens, int32_t n_q,
                              int32_t n_kv, int32_t head_dim, void* out, int32_t* work_queues, void* stream) {
  if (!work_queues) return guarded(nullptr, [&] { fail(MZ_EINVAL, "work_queues is NULL"); });
  return attention_entry(q, qpos, m, slab, table, n_table, chunk_tokens, n_q, n_kv, head_dim, out, work_queues,
                         stream);
}

int64_t mz_attention_split_workspace_bytes(int32_t m, int32_t n_q, int32_t head_dim, int32_t n_split) {
  if (m < 1 || n_q < 1 || (head_dim != 64 && head_dim != 128) || n_split < 1) return -1;
  return mzk::attention_split_ws_bytes(m, n_q, head_dim, n_split);
}

int32_t mz_attention_auto_splits(int32_t m, int32_t max_pos, int32_t n_q, int32_t n_kv, int32_t head_dim,
                                 int64_t workspace_bytes) {
  if (m < 1 || max_pos < 0 || n_kv < 1 || n_q % n_kv || (head_dim != 64 && head_dim != 128)) return 1;
  return mzk::attention_auto_splits(m, max_pos, n_q, n_kv, head_dim, workspace_bytes);
}

mz_status mz_attention_split(const void* q, const int32_t* qpos, int32_t m, int32_t max_pos, const void* slab,
                             const int32_t* table, int32_t n_table, int32_t chunk_tokens, int32_t n_q,
                             int32_t n_kv, int32_t head_dim, int32_t n_split, void* workspace,
                             int64_t workspace_bytes, void* out, void* stream) {
  return guarded(nullptr, [&] {
    if (!q || !qpos || !slab || !table || !out || !workspace) fail(MZ_EINVAL, "NULL pointer");
    if (m < 1 || n_table < 1 || max_pos < 0) fail(MZ_EINVAL, "sizes must be positive");
    if (n_table > mzk::kAttnTableMax) fail(MZ_EINVAL, "n_table above %d", mzk::kAttnTableMax);
    if (chunk_tokens < 8 || (chunk_tokens & (chunk_tokens - 1))) fail(MZ_EINVAL, "chunk_tokens must be a power of two >= 8");
    if (head_dim != 64 && head_dim != 128) fail(MZ_EINVAL, "head_dim must be 64 or 128");
    if (n_kv < 1 || n_q % n_kv || n_q / n_kv > 8) fail(MZ_EINVAL, "bad head counts");
    if (max_pos / chunk_tokens >= n_table) fail(MZ_EINVAL, "table does not cover max_pos");
    if (n_split < 1 || n_split > 64) fail(MZ_EINVAL, "n_split must be 1..64");
    if (workspace_bytes < mzk::attention_split_ws_bytes(m, n_q, head_dim, n_split))
      fail(MZ_EINVAL, "workspace too small for %d splits", n_split);
    const int64_t slot_bytes = (int64_t)chunk_tokens * n_kv * head_dim * 2 * 2;
    mzk::launch_attention_split(q, qpos, m, max_pos, slab, table, n_table, chunk_tokens, slot_bytes, n_q, n_kv, head_dim,
                                n_split, workspace, out, (hipStream_t)stream);
    HIPCHK(hipGetLastError());
  });
}

mz_status mz_rmsnorm(const void* h, int32_t m, int32_t d, float eps, void* x, void* stream) {
  return guarded(nullptr, [&] {
    if (!h || !x) fail(MZ_EINVAL, "NULL pointer");
    if (m < 1 || d < 4 || d % 4) fail(MZ_EINVAL, "bad sizes");
    mzk::launch_rmsnorm((const float*)h, m, d, eps, x, (hipStream_t)stream);
    HIPCHK(hipGetLastError());
  });
}

mz_status mz_kv_compress(const void* src, int64_t n_halves, void* out, void* stream) {
  return guarded(nullptr, [&] {
    if (!src || !out) fail(MZ_EINVAL, "NULL pointer");
    if (n_halves < 64 || n_halves % 64) fail(MZ_EINVAL, "n_halves must be a positive multiple of 64");
    mzk::launch_kv_compress(src, nullptr, 0, n_halves, 1, out, (hipStream_t)stream);
    HIPCHK(hipGetLastError());
  });
}

mz_status mz_kv_decompress(const void* in, int64_t n_halves, void* dst, void* stream) {
  return guarded(nullptr, [&] {
    if (!in || !dst) fail(MZ_EINVAL, "NULL pointer");
    if (n_halves < 64 || n_halves % 64) fail(MZ_EINVAL, "n_halves must be a positive multiple of 64");
    mzk::launch_kv_decompress(in, n_halves, 1, dst, nullptr, 0, (hipStream_t)stream);
    HIPCHK(hipGetLastError());
  });
}

mz_status mz_probe_ceilings(int32_t device, char* json_out, size_t cap) {
  return guarded(nullptr, [&] {
    if (!json_out || cap < 2) fail(MZ_EINVAL, "json_out is NULL or too small");
    HIPCHK(hipSetDevice(device));
    hipStream_t s = nullptr;
    HIPCHK(hipStreamCreateWithFlags(&s, hipStreamNonBlocking));
    hipEvent_t e0 = nullptr, e1 = nullptr;
    float* out = nullptr;
    void *a = nullptr, *b = nullptr, *host = nullptr;
    auto cleanup = [&] {
      if (out) (void)hipFree(out);
      if (a) (void)hipFree(a);
      if (b) (void)hipFree(b);
      if (host) (void)hipHostFree(host);
      if (e0) (void)hipEventDestroy(e0);
      if (e1) (void)hipEventDestroy(e1);
      if (s) (void)hipStreamDestroy(s);
    };
    try {
      HIPCHK(hipEventCreate(&e0));
      HIPCHK(hipEventCreate(&e1));
      // best of a few timed runs of f(), in ms
      auto best_ms = [&](int reps, auto&& f) {
        float best = 1e30f;
        f();   // warm-up (clocks, code load)
        for (int r = 0; r < reps; ++r) {
          HIPCHK(hipEventRecord(e0, s));
          f();
          HIPCHK(hipEventRecord(e1, s));
          HIPCHK(hipEventSynchronize(e1));
          float ms = 0;
          HIPCHK(hipEventElapsedTime(&ms, e0, e1));
          best = std::min(best, ms);
        }
        return (double)best;
      };
      const int blocks = 2048, iters = 16000;   // ~45 ms per run: long enough for the clock to settle
      HIPCHK(hipMalloc((void**)&out, (size_t)blocks * 512 * sizeof(float)));
      double tf[3];
      for (int mode = 0; mode < 3; ++mode) {
        const double ms = best_ms(3, [&] { mzk::launch_mfma_probe(out, blocks, iters, mode, s); });
        tf[mode] = mzk::mfma_probe_flops_per_launch(blocks, iters) / (ms * 1e-3) / 1e12;
      }
      const size_t bytes = (size_t)1 << 30;
      HIPCHK(hipMalloc(&a, bytes));
      HIPCHK(hipMalloc(&b, bytes));
      mzk::launch_fill(a, bytes / 4, 0x3C003C00u, s);
      const double copy_ms = best_ms(3, [&] { mzk::launch_copy_probe(a, b, (int64_t)bytes, s); });
      HIPCHK(hipHostMalloc(&host, bytes, hipHostMallocDefault));
      memset(host, 1, bytes);
      const double h2d_ms = best_ms(3, [&] { HIPCHK(hipMemcpyAsync(a, host, bytes, hipMemcpyHostToDevice, s)); });
      const double d2h_ms = best_ms(3, [&] { HIPCHK(hipMemcpyAsync(host, b, bytes, hipMemcpyDeviceToHost, s)); });
      HIPCHK(hipStreamSynchronize(s));
      char buf[512];
      snprintf(buf, sizeof buf,
               "{\"mfma_f16_tflops\": %.1f, \"mfma_f16_codes_tflops\": %.1f, "
               "\"mfma_f16_block_scaled_tflops\": %.1f, \"hbm_copy_gbps\": %.1f, \"h2d_pinned_gbps\": %.2f, "
               "\"d2h_pinned_gbps\": %.2f}",
               tf[0], tf[1], tf[2], 2.0 * bytes / (copy_ms * 1e-3) / 1e9, bytes / (h2d_ms * 1e-3) / 1e9,
               bytes / (d2h_ms * 1e-3) / 1e9);
      if (strlen(buf) + 1 > cap) fail(MZ_EINVAL, "json_out buffer too small");
      memcpy(json_out, buf, strlen(buf) + 1);
    } catch (...) {
      cleanup();
      throw;
    }
    cleanup();
  });
}

}  // extern "C"
