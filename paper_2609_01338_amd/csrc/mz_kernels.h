// Launchers of the gfx950 kernels of the restore-and-prefill path.  Each takes
// device pointers and a stream, checks nothing, and enqueues one kernel; the
// callers (runtime and ABI) validate shapes first.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mzk {

// Device GEMM layout of a Q4_0 matrix [n][k]: tiles of 256 rows x 64 columns,
// ordered n-tile major, k-tile minor.  A tile holds 256*2 blocks of 16 nibble
// bytes (row-major over (row, block)), then their 256*2 fp16 scales.  Within
// a block the 32 codes are re-ordered: dword i carries elements 8i..8i+7 with
// element 8i+2m at bits 4m..4m+3 and element 8i+2m+1 at bits 16+4m..19+4m.
constexpr int kGemmTileN = 256;
constexpr int kGemmTileK = 64;
constexpr int kGemmTileBytes = kGemmTileN * kGemmTileK / 2 + kGemmTileN * (kGemmTileK / 32) * 2;

enum GemmEpilogue { kEpiStore = 0, kEpiAdd = 1, kEpiSwiGLU = 2, kEpiPartial = 3, kEpiRopeQ = 4, kEpiRopeKV = 5 };

// Rotary-embedding epilogues (rotate-half pairs c, c + hd/2 of each head at
// the row's position, (cos, sin) from rope_cs [pos][hd/2], rounded to f16).
// kEpiRopeQ: y f16 [m][n_valid] holds the rotated queries (n_valid = q
// columns).  kEpiRopeKV: output columns [0, n_valid/2) are keys, rotated and
// written to slab + kv_off[r] (the row's token-major K row of its chunk
// slot); [n_valid/2, n_valid) are values, written to the slot's V^T half
// (V^T[c][pos % C] at slot + C * (n_valid/2) * 2 + (c * C + pos % C) * 2);
// rows with kv_off < 0 write nothing.  pos is indexed by output row.
struct GemmRope {
  const int32_t* pos = nullptr;
  const int64_t* kv_off = nullptr;
  const float2* rope_cs = nullptr;
  uint8_t* slab = nullptr;
  int hd = 0, n_valid = 0, C = 0;
};

// Y = X . W^T: X f16 [m][k], W packed [n][k] (n % 128 == 0, k % 64 == 0).
// kEpiStore: Y float [m][n] = acc; kEpiAdd: Y float [m][n] += acc;
// kEpiSwiGLU: Y f16 [m][n/2] = silu(gate) * up for the interleaved layout.
// With a_rows (device, m entries), output row r is computed from X row a_rows[r].
// With work_queues (device, kGemmQueueInts int32, zero on entry and left zero
// on return; not shared by launches in flight together), persistent
// workgroups take the tiles from per-XCD queues, so XCDs that run faster take
// more of them; the results are the same bits.  (launch_gemm_q4_rope takes
// the argument but always runs one workgroup per tile.)
constexpr int kGemmQueueInts = 16;
// With ws (ws_bytes of device scratch, not in use by launches in flight), a
// ragged remainder of rows whose tiles alone would leave most CUs idle runs
// split over K (as launch_gemm_q4_splitk) instead of as 64-row tiles, and a
// product whose 256-row tiles are too few for the chip but whose K range is
// long runs as 256-row tiles split over K (gemm_long_k_splits) instead of as
// 64-row tiles over the whole K range.
void launch_gemm_q4(const void* x, int m, int n, int k, const void* w, int epilogue, void* y,
                    hipStream_t s, const int32_t* a_rows = nullptr, int* work_queues = nullptr,
                    void* ws = nullptr, int64_t ws_bytes = 0);

// Y = X . W^T with a rotary-embedding epilogue (kEpiRopeQ / kEpiRopeKV, see
// GemmRope); n_valid <= n.  Only for gemm_rope_fusable(hd, C): head
// dimension 32, 64 or 128, C a power of two.
bool gemm_rope_fusable(int head_dim, int chunk_tokens);
void launch_gemm_q4_rope(const void* x, int m, int n, int k, const void* w, int epilogue, const GemmRope& ea,
                         void* y, hipStream_t s, const int32_t* a_rows = nullptr, int* work_queues = nullptr,
                         void* ws = nullptr, int64_t ws_bytes = 0);

// Split-K form for few rows: n_split ranges of whole 64-wide K steps
// (ceil((k / 64) / n_split) steps each) write fp32 partials into ws
// (gemm_splitk_ws_bytes(m, n, n_split) bytes), then one kernel adds them in
// split order and applies the epilogue.  h_norm (m == 1 only): x is not read;
// the row is RMSNorm(h_norm row, eps) formed inside the product, the same
// f16 values launch_rmsnorm writes.  row_tile: 64 or 256 rows per partial
// tile (0: the size launch_gemm_q4 takes for m rows).
void launch_gemm_q4_splitk(const void* x, int m, int n, int k, const void* w, int epilogue, void* y, int n_split,
                           void* ws, hipStream_t s, const int32_t* a_rows = nullptr,
                           const float* h_norm = nullptr, float eps = 0.f, int row_tile = 0);
int64_t gemm_splitk_ws_bytes(int m, int n, int n_split);
// Split-K form with a rotary-embedding epilogue (kEpiRopeQ / kEpiRopeKV): the
// splits are added in order, then rotated and written as the unsplit
// epilogues do.
void launch_gemm_q4_splitk_rope(const void* x, int m, int n, int k, const void* w, int epilogue, const GemmRope& ea,
                                void* y, int n_split, void* ws, hipStream_t s, const int32_t* a_rows = nullptr,
                                const float* h_norm = nullptr, float eps = 0.f, int row_tile = 0);
// One activation row in one launch (m = 1, no workspace): workgroups own a
// few output columns over the whole K range and apply the epilogue
// themselves (any of kEpiStore .. kEpiRopeKV, with ea as for
// launch_gemm_q4_rope).  The code-activation products are exact and each
// block's scale multiplies its fp32 sum (no f16 rounding of d (q - 8)).  h_norm as in launch_gemm_q4_splitk.  Only where
// gemv1_ok(n, k): n % 256 == 0, k % 64 == 0, k <= kGemv1MaxK (the row is
// staged in LDS).
constexpr int kGemv1MaxK = 16384;
bool gemv1_ok(int n, int k);
void launch_gemv1(const void* x, int n, int k, const void* w, int epilogue, const GemmRope& ea, void* y,
                  hipStream_t s, const int32_t* a_rows = nullptr, const float* h_norm = nullptr, float eps = 0.f);
// The rotary query product (kEpiRopeQ into yq, eq) and the key/value product
// into the chunk slot (kEpiRopeKV, ekv) of one row in one launch, both of k
// inputs from x (or RMSNorm(h_norm)); the same results as the two
// launch_gemv1 calls.  Only where gemv1_ok holds for both.
void launch_gemv1_qkv(const void* x, int k, const void* wq, void* yq, const GemmRope& eq, const int32_t* rows_q,
                      const void* wkv, const GemmRope& ekv, const int32_t* rows_kv, hipStream_t s,
                      const float* h_norm = nullptr, float eps = 0.f);
// Splits that fill the chip for this shape within ws_cap bytes (1: no split).
int gemm_auto_splits(int m, int n, int k, int64_t ws_cap);
// K splits of 256-row tiles for launch_gemm_q4 with a workspace of ws_cap
// bytes where its 256-row tiles alone are too few for the chip, the 64-row
// tiles fill it and every split keeps at least 16 K steps; 1 otherwise.
int gemm_long_k_splits(int m, int n, int k, int64_t ws_cap);

// Causal GQA attention over chunked KV (see mz.h, mz_attention).  table has
// n_table entries (at most kAttnTableMax).  With
// work_queues (device, kAttnQueueInts int32, zero on entry and left zero on
// return; not shared by launches in flight together) and n_kv dividing 8,
// persistent workgroups take the query tiles from per-KV-head queues, so
// XCDs that run faster take more of them; otherwise one workgroup per tile.
constexpr int kAttnQueueInts = 16;
constexpr int kAttnTableMax = 8192;
void launch_attention(const void* q, const int32_t* qpos, int m, const void* slab,
                      const int32_t* table, int n_table, int chunk_tokens, int64_t slot_bytes, int n_q,
                      int n_kv, int head_dim, void* out, hipStream_t s, int* work_queues = nullptr);

// Split-key attention for few query rows: n_split key ranges of whole 64-key
// tiles (tiles per split = ceil((max_pos / 64 + 1) / n_split)) run as separate
// workgroups writing partials into ws, then a merge kernel writes out.
// max_pos >= qpos[m - 1]; ws holds attention_split_ws_bytes(m, n_q,
// head_dim, n_split) bytes.
void launch_attention_split(const void* q, const int32_t* qpos, int m, int max_pos, const void* slab,
                            const int32_t* table, int n_table, int chunk_tokens, int64_t slot_bytes, int n_q,
                            int n_kv, int head_dim, int n_split, void* ws, void* out, hipStream_t s);
int64_t attention_split_ws_bytes(int m, int n_q, int head_dim, int n_split);
// Splits that fill the chip for this shape within ws_cap bytes (1: no split).
int attention_auto_splits(int m, int max_pos, int n_q, int n_kv, int head_dim, int64_t ws_cap);

// x f16 [m][d] = RMSNorm(h float [m][d]).
void launch_rmsnorm(const float* h, int m, int d, float eps, void* x, hipStream_t s);

// Rotary embedding + KV scatter.  qkv float [m][qkv_stride] holding nq query
// heads, then nkv key heads and nkv value heads (either group may be empty);
// rope_cs float2 [max_pos][hd/2] (cos, sin); kv_off int64 [m] (may be null when
// nkv is 0): byte offset in slab of the row's K (token-major [C][dkv] slot
// half) or -1 to skip; the row's V goes to the slot's V^T half ([dkv][C]).
// q_out f16 [m][nq*hd].  C is a power of two.
void launch_rope_kv(const float* qkv, int qkv_stride, int m, const int32_t* pos,
                    const int64_t* kv_off, const float2* rope_cs, int nq, int nkv, int hd, int C,
                    void* q_out, void* slab, hipStream_t s);

// h float [m][d] = dequant(E[tok[i]]) with E split into nibbles [V][d/2] and
// fp16 scales [V][d/32]; with last_tok (device) row m - 1 takes *last_tok.
void launch_embed(const uint8_t* e_nib, const uint16_t* e_scale, const int32_t* tok, int m, int d,
                  float* h, hipStream_t s, const int32_t* last_tok = nullptr);

// dst[i] = src[idx[i]] for rows of d floats.
void launch_gather_rows(const float* src, const int32_t* idx, int m, int d, float* dst,
                        hipStream_t s);

// logits float [V] = RMSNorm(h_last) . W_lm^T (split layout as the embedding),
// then token = argmax (lowest index on ties), also stored to token2 when
// given.  part_val/part_idx hold ceil(V / 256) partials (256 rows a block).
void launch_lm_head(const float* h_last, int d, float eps, const uint8_t* w_nib,
                    const uint16_t* w_scale, int vocab, float* logits, float* part_val,
                    int32_t* part_idx, int32_t* token, hipStream_t s, int32_t* token2 = nullptr);

// Fill n 32-bit words with zero (graph-capturable, unlike memset nodes).
void launch_zero(void* p, int64_t n_words, hipStream_t s);

// Fill n 32-bit words with `value` (test hook: NaN-poison fresh slots).
void launch_fill(void* p, int64_t n_words, uint32_t value, hipStream_t s);

// Busy-wait about `us` microseconds of wall clock on stream s (test hook that
// delays a stream).  Bounded: always exits.
void launch_spin(int64_t us, hipStream_t s);

// Ceiling probes: blocks x 512 threads of f16 MFMAs with changing operands
// (out: blocks*512 floats; mode 0 random halves, 1 the B operand as exact
// 4-bit codes, 2 codes with each 32-deep product scaled into the sum by
// fp32 FMAs), and a plain copy of `bytes` (multiple of 16).
double mfma_probe_flops_per_launch(int blocks, int iters);
void launch_mfma_probe(float* out, int blocks, int iters, int mode, hipStream_t s);
void launch_copy_probe(const void* src, void* dst, int64_t bytes, hipStream_t s);

// 8-bit group-wise KV codec (groups of 64 halves; compressed run = n code
// bytes, then (min, step) halves per group).  n_runs runs of n_halves each:
// run r is read from src_base + (src_slots ? src_slots[r] : r) * src_stride
// and written to dst + r * kv_compressed_bytes(n_halves); decompression the
// other way round (dst_base + (dst_slots ? dst_slots[r] : r) * dst_stride).
int64_t kv_compressed_bytes(int64_t n_halves);
void launch_kv_compress(const void* src_base, const int32_t* src_slots, int64_t src_stride, int64_t n_halves,
                        int n_runs, void* dst, hipStream_t s);
void launch_kv_decompress(const void* src, int64_t n_halves, int n_runs, void* dst_base,
                          const int32_t* dst_slots, int64_t dst_stride, hipStream_t s);

}  // namespace mzk
