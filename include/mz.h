/*
 * mz.h -- C ABI of the MI355X restore-and-prefill engine.
 *
 * The engine rebuilds an evicted LLM context on one GPU.  The model's weights
 * are held per transformer layer and its KV cache per layer in fixed-size
 * token chunks (paper Sec. 4.2); each unit is resident, swapped to pinned host
 * memory, or dropped.  Restoring copies swapped units back and recomputes
 * dropped KV chunks with a Q4_0-weight Llama-style prefill, layer by layer, so
 * the first token waits only for what is actually missing.  The calls follow
 * the paper's interface pair evict(size) / restore_generate(input_tokens)
 * (Sec. 5), with the eviction amount given as an explicit per-unit plan.
 *
 * Conventions shared by every call:
 *  - Every call returns mz_status.  On error the context is left as it was
 *    and mz_last_error() describes the failure.
 *  - The library owns all device memory and all pinned host memory it
 *    allocates.  Input arrays are copied before the call returns; the caller
 *    owns every output buffer.
 *  - "host" pointers are ordinary CPU memory; "device" pointers are HBM
 *    addresses on the context's GPU (the kernel-level calls at the end).
 *  - One context is used by one thread at a time.
 */
#ifndef MZ_H
#define MZ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct mz_ctx mz_ctx;

typedef enum {
  MZ_OK = 0,
  MZ_EINVAL = -1,   /* bad shape, token id, state value or size */
  MZ_ENOMEM = -2,   /* pool, arena or device allocation exhausted */
  MZ_EHIP = -3,     /* a HIP runtime call failed */
  MZ_ESTATE = -4    /* call not valid in the current state */
} mz_status;

/* State of one unit (a layer's weights, or one KV chunk of one layer). */
typedef enum { MZ_RES = 0, MZ_SWAP = 1, MZ_DROP = 2 } mz_unit_state;

/* Model shape.  d_model must be a multiple of 256, at most 8192; d_ffn need not be a
 * multiple of 32 (Q4_0 rows of W_down are zero-padded); head_dim must be 64 or
 * 128; n_q_heads a multiple of n_kv_heads with a group of at most 8;
 * chunk_tokens a power of two (>= 8); max_ctx bounds context + prompt tokens. */
typedef struct {
  int32_t n_layers, d_model, n_q_heads, n_kv_heads, head_dim, d_ffn, vocab;
  int32_t chunk_tokens, max_ctx;
  float rope_theta, rms_eps;
} mz_model_cfg;

/* Eviction plan (paper Sec. 4.3-4.4).  kv_state is [n_layers][n_chunks]
 * (n_chunks = chunks of the cached context), w_state is [n_layers] or NULL
 * (all resident).  A target of MZ_RES leaves a unit as it is; MZ_SWAP moves a
 * resident unit to the pinned host arena; MZ_DROP releases it (a dropped KV
 * chunk is recomputed at restore; a dropped weight unit is reloaded from the
 * model image kept in host memory, standing in for the paper's storage).
 * Units are visited in `order` (unit ids: KV chunk (l, c) is l * n_chunks + c,
 * weight unit l is n_layers * n_chunks + l); NULL means backward-out: last
 * layer first, within a layer its chunks from the last, then its weights
 * (Sec. 4.4).  Swapped units are pushed on the arena stack in that order. */
typedef struct {
  const uint8_t *kv_state;
  int32_t n_layers;
  int32_t n_chunks;
  const uint8_t *w_state;
  const int32_t *order;
  int32_t n_order;
} mz_evict_plan;

/* ---- model-level calls ------------------------------------------------- */

/* Create a context on GPU `device` from a Q4_0 model blob (host, nbytes).
 * Blob: per layer Wq, Wk, Wv, Wo, W_gate, W_up, W_down, then E and W_lm; each
 * [out][in] as rows of ceil(in/32) 18-byte Q4_0 blocks (fp16 scale, then 16
 * bytes: element j in the low nibble of byte j, element j+16 in the high).
 * The blob is repacked into device layouts and a host copy of the layer
 * weights is retained for dropped-weight reloads.  EINVAL on a shape or size
 * mismatch or more than 8192 chunks per layer (max_ctx / chunk_tokens),
 * ENOMEM / EHIP on allocation failure. */
mz_status mz_load_model(const mz_model_cfg *cfg, const void *q4_blob, size_t nbytes,
                        int32_t device, mz_ctx **out);

/* Replace the cached context by tokens[0..n) (host) and build its KV cache
 * with a full prefill on the GPU: every layer computes the key and value
 * vectors of every token, kept as the KV cache (paper Sec. 2.1), here in the
 * per-layer chunk slots (Sec. 4.2); every chunk is resident afterwards.
 * EINVAL for n < 0, n > max_ctx, a NULL tokens with n > 0, or a token id
 * outside the vocabulary. */
mz_status mz_prefill_context(mz_ctx *ctx, const int32_t *tokens, int32_t n);

/* Replace the cached context by tokens[0..n) (host) without computing KV:
 * every chunk is allocated, zero-filled and resident; fill it with
 * mz_import_kv.  Used to start from KV produced elsewhere -- the cached
 * context of a context-aware request (paper Sec. 2.2) whose KV cache was
 * built before.  Errors as mz_prefill_context. */
mz_status mz_set_context(mz_ctx *ctx, const int32_t *tokens, int32_t n);

/* Write chunk `chunk` of layer `layer` -- one KV unit of the fine-grained
 * memory management, a fixed run of tokens of one layer's K and V (paper
 * Sec. 4.2, chunk size in Sec. 4.3) -- from host arrays k, v, each
 * [chunk_tokens][n_kv_heads * head_dim] IEEE half, hidden index innermost
 * (the exchange layout; the device slot keeps V transposed).  Rows past the
 * context's last token are written too.  EINVAL for a layer or chunk out of
 * range, ESTATE if the chunk is not resident. */
mz_status mz_import_kv(mz_ctx *ctx, int32_t layer, int32_t chunk, const void *k_f16,
                       const void *v_f16);

/* Read a resident KV chunk (paper Sec. 4.2) into host arrays k, v laid out
 * as in mz_import_kv (caller-owned, chunk_tokens * n_kv_heads * head_dim
 * halves each).  EINVAL for a layer or chunk out of range, ESTATE if the
 * chunk is not resident. */
mz_status mz_read_kv(mz_ctx *ctx, int32_t layer, int32_t chunk, void *k_f16, void *v_f16);

/* Keep only the first n tokens of the cached context (0 <= n <= current):
 * chunks entirely past n are released and the rest stay as they are.  Every
 * unit must be resident (ESTATE otherwise). */
mz_status mz_truncate_context(mz_ctx *ctx, int32_t n);

/* Apply an eviction plan (idle phase; synchronous).  Allowed moves:
 * RES->SWAP, RES->DROP, SWAP->DROP.  ESTATE for SWAP of a dropped unit or when
 * no context is cached; EINVAL for a plan whose shape does not match. */
mz_status mz_evict(mz_ctx *ctx, const mz_evict_plan *plan);

/* Restore every evicted unit and prefill prompt[0..n_prompt) (host) after the
 * cached context.  Swapped units are copied back on a side stream earliest
 * layer first (forward-in, Sec. 4.4) while the compute stream recomputes the
 * dropped chunks; each layer's compute waits only on that layer's copies.
 * Asynchronous: returns once the work is enqueued.  Afterwards every unit is
 * resident and the context holds n_ctx + n_prompt tokens.  EINVAL if the
 * total exceeds max_ctx or a token is out of range. */
mz_status mz_restore_and_prefill(mz_ctx *ctx, const int32_t *prompt, int32_t n_prompt);

/* Greedy first token after mz_restore_and_prefill / mz_prefill_context --
 * the token that ends the prefill stage, whose latency is the TTFT (paper
 * Sec. 2.1): RMSNorm of the last position's final hidden state, output head,
 * argmax (lowest index on ties).  Synchronizes.  logits_out (host, [vocab]
 * float) may be NULL.  EINVAL for a NULL token_out, ESTATE if nothing was
 * prefilled since the last first token. */
mz_status mz_first_token(mz_ctx *ctx, int32_t *token_out, float *logits_out);

/* Greedy generation past the first token: append `token` to the context,
 * run it through every layer (one row; its attention reads the whole
 * context, split over the keys), take the argmax of its logits as
 * tokens_out[0]; then append that and continue, n tokens in all (host,
 * caller-owned tokens_out [n]).  The last generated token is not appended,
 * as with mz_first_token.  Any evicted units are restored by the first step
 * (it is a restore with a one-token prompt).  The steps after the first are
 * issued back to back: each step's token stays on the device for the next
 * step's embedding, and tokens_out is written when all have run.  Errors:
 * EINVAL (n < 0, NULL tokens_out, token out of range, or a context that
 * would pass max_ctx), and those of mz_restore_and_prefill; tokens_out then
 * holds the tokens of the steps that ran. */
mz_status mz_generate(mz_ctx *ctx, int32_t token, int32_t n, int32_t *tokens_out);

/* Engine options: "overlap" (1: swap-in overlapped with compute, default;
 * 0: every copy finishes before compute starts), "kernel_timing" (1: time
 * every kernel launch with HIP events on its stream; setting it clears the
 * accumulated kernel statistics), "kv_codec" (1: mz_evict compresses every
 * full swapped KV chunk with the 8-bit codec of mz_kv_compress and restores
 * it through mz_kv_decompress -- about half the host-link bytes, values
 * rounded to the codec's grid; partial chunks and weight units move raw;
 * enabling it the first time allocates a device staging ring of one layer's
 * chunks), "attn_split" (1: attention of few query rows against a long
 * context runs split over the keys, as mz_attention_split, default; 0: always
 * one pass), "attn_queue" (1: the attention of many rows, at least
 * 4 * 256 (query row, query head) pairs per compute unit, runs as
 * mz_attention_queued with queues owned by the context, default; 0: as
 * mz_attention), "gemm_queue" (1: the unsplit projections with a store,
 * residual-add or SwiGLU epilogue run as mz_q4_gemm_queued, default; 0: one
 * workgroup per tile), "gemm_split" (1: GEMMs of few rows run split over K, as
 * mz_q4_gemm_split, default; 0: never), "fuse_rope" (1: the query and
 * key/value projections apply the rotary embedding in their epilogue, or in
 * the reduce of their K splits, and write f16 queries and the chunk slots
 * directly, default; 0: projection, then a separate RoPE pass), "fuse_norm"
 * (1: a layer step of a single row whose projections all run split over K
 * forms that row's RMSNorm inside them, the same f16 values the RMSNorm
 * pass writes, and leaves that pass out, default; 0: always a separate
 * pass), "swap_trim" (1: free the pinned swap segments after each restore,
 * as the paper's growing swap stack does; 0: keep them for the next
 * eviction, default).  Test hooks: "debug_poison" (1: fill every
 * slot and weight unit allocated by a restore with NaN before it is
 * restored or recomputed), "debug_swap_delay_us" (delay the swap stream by a
 * bounded busy wait before its copies), "debug_kv_slot_limit" (at most this
 * many KV chunk slots in use, so a restore that needs more fails with
 * MZ_ENOMEM and leaves the context as it was; negative: the whole pool, the
 * default).  EINVAL for an unknown key. */
mz_status mz_set_option(mz_ctx *ctx, const char *key, int64_t value);

/* JSON summary of the last restore (row counts, bytes moved, per-kernel
 * launch counts / time / algorithmic work, pool occupancy), written to
 * json_out (host, cap bytes, NUL-terminated).  EINVAL if cap is too small. */
mz_status mz_stats(mz_ctx *ctx, char *json_out, size_t cap);

/* Description of the last error on ctx (or of the last failed mz_load_model
 * when ctx is NULL).  Valid until the next call on the same context. */
const char *mz_last_error(const mz_ctx *ctx);

/* Release the context and everything it owns (NULL is allowed). */
void mz_free(mz_ctx *ctx);

/* ---- host-only helpers (no GPU needed) --------------------------------- */

/* Library version string. */
const char *mz_version(void);

/* Rows of the restore (R_l: positions that pass through layer l; D_l: rows
 * whose layer-l K/V is written) for kv_state [n_layers][n_chunks] (host),
 * n_ctx context and n_prompt prompt tokens.  Writes nR[l], nD[l] (host,
 * [n_layers]) and, if rows is not NULL, the concatenation of every R_l
 * (ascending positions) into rows (host, rows_cap entries).  EINVAL if
 * rows_cap is too small. */
mz_status mz_plan_rows(const mz_model_cfg *cfg, const uint8_t *kv_state, int32_t n_chunks,
                       int32_t n_ctx, int32_t n_prompt, int32_t *nR, int32_t *nD,
                       int32_t *rows, int64_t rows_cap);

/* ---- eviction planning (host only) ------------------------------------ */

/* Order in which units are evicted (paper Sec. 4.4 for backward-out). */
typedef enum {
  MZ_ORDER_BACKWARD_OUT = 0,   /* layer descending, chunk descending */
  MZ_ORDER_FORWARD_OUT = 1,    /* layer ascending, chunk ascending */
  MZ_ORDER_RANDOM_OUT = 2,     /* uniform shuffle (Fisher-Yates driven by splitmix64(seed)) */
  MZ_ORDER_TOKEN_ALIGNED = 3   /* chunk column descending, all layers of a column together */
} mz_evict_order;

/* Restore path of each evicted KV chunk. */
typedef enum {
  MZ_PLACE_BALANCED = 0,       /* each chunk to the path that keeps max(link, recompute) time smallest */
  MZ_PLACE_ALL_SWAP = 1,
  MZ_PLACE_ALL_DROP = 2,
  MZ_PLACE_INTERLEAVE_2_1 = 3  /* rank r in the order dropped iff r mod 3 = 2 */
} mz_placement;

typedef struct {
  int32_t n_ctx;               /* cached tokens; chunks per layer = ceil(n_ctx / chunk_tokens) */
  int32_t n_prompt;            /* prompt tokens of the coming restore (they enter the work model) */
  int32_t n_kv_evict;          /* KV chunks to evict, the first ones of `order` */
  int32_t n_w_evict;           /* weight units to evict (always swapped): the last layers, the
                                  first for MZ_ORDER_FORWARD_OUT */
  int32_t order;               /* mz_evict_order */
  int32_t placement;           /* mz_placement */
  uint64_t seed;               /* MZ_ORDER_RANDOM_OUT */
  double link_bytes_per_s;     /* host link rate (MZ_PLACE_BALANCED) */
  double recompute_flops_per_s;/* effective recompute rate (MZ_PLACE_BALANCED) */
  int32_t kv_codec;            /* 1: full chunks cross the link compressed (option "kv_codec") */
} mz_evict_request;

/* Eviction plan for mz_evict: the paper's hybrid-swap balance (Sec. 4.3)
 * re-targeted to this engine's two restore paths, the host link (weights and
 * KV chunks) and GPU recompute (KV chunks), with its forward-in restore
 * (Sec. 4.4).  The balanced placement walks the evicted KV chunks in order
 * and gives each to the path that finishes the restore earlier under the
 * restore's schedule: units arrive over the link layer by layer, and layer
 * l computes once layer l-1 is done and layer l's units have arrived, its
 * work being the restore's exact FLOP count for the plan so far (dropping a
 * chunk at layer l pulls its rows through every layer <= l, so its cost
 * depends on the rest of the plan).  Outputs (host, caller-owned):
 * kv_state [n_layers][ceil(n_ctx / chunk_tokens)], w_state [n_layers]
 * (MZ_RES / MZ_SWAP / MZ_DROP), and est (NULL or 5 doubles: swapped bytes,
 * restore FLOPs, link seconds, recompute seconds, and the schedule's finish
 * time in seconds; the times need both rates).  Errors: EINVAL (sizes,
 * unknown order or placement, non-positive rates for the balanced placement). */
mz_status mz_plan_evict(const mz_model_cfg *cfg, const mz_evict_request *req, uint8_t *kv_state,
                        uint8_t *w_state, double *est);

/* ---- size-driven eviction (host planning + mz_evict) ------------------ */

/* Stage of the hybrid-swap eviction policy (paper Sec. 4.3, Alg. 1). */
typedef enum {
  MZ_STAGE_KV_ONLY = 0,        /* KV chunks only, each to the path that keeps both totals level */
  MZ_STAGE_KV_AND_W = 1,       /* weight layers, with the KV chunks their reload time covers dropped */
  MZ_STAGE_W_ONLY = 2,         /* weight layers only (no KV chunk left) */
  MZ_STAGE_EXHAUSTED = 3       /* nothing resident is left to evict */
} mz_evict_stage;

/* How the threshold T and the KV_AND_W pairing are formed (see mz_plan_evict_size). */
typedef enum {
  MZ_SIZE_RULE_PAPER = 0,      /* T = N_W^total * floor(t_W / t_d), floor(t_W / t_d) chunks per weight layer */
  MZ_SIZE_RULE_TOTAL = 1       /* T and the pairing from the path totals of the plan's exact costs */
} mz_size_rule;

typedef struct {
  int64_t bytes;               /* device bytes to release: KV slots and weight units */
  int32_t n_prompt;            /* expected prompt length of the coming restore (0 if unknown) */
  int32_t n_w_total;           /* evictable weight layers N_W^total (the last ones), 0..n_layers */
  double link_bytes_per_s;     /* host link rate */
  double recompute_flops_per_s;/* GPU recompute rate */
  int32_t kv_codec;            /* 1: full swapped chunks are priced at their compressed size */
  int32_t rule;                /* mz_size_rule (0, the paper's, in a zeroed request) */
} mz_evict_size_request;

/* Plan the next increment of size-driven eviction from the current unit
 * states (the paper's evict(size), Sec. 5, driven by its hybrid-swap policy,
 * Sec. 4.3 and Alg. 1, and its backward-out order, Sec. 4.4).  The two
 * restore paths are the host link (weight layers and swapped KV chunks: a
 * unit costs its link bytes / link rate) and GPU recompute (dropped KV
 * chunks: a chunk costs the growth of the restore's exact FLOP count when it
 * is dropped, / recompute rate; this depends on the rest of the plan).
 * Totals: link = every non-resident weight unit and swapped chunk, recompute
 * = FLOPs(plan) - FLOPs(nothing dropped).  N_KV and N_W count the resident
 * chunks and evictable weight layers.  Threshold and pairing (req->rule):
 *   MZ_SIZE_RULE_PAPER  the paper's (Sec. 4.3): t_W = one weight unit's link
 *                       time, t_d = the recompute time of the front-most chunk
 *                       (chunk 0 of layer 0, restored last in backward-out
 *                       order) dropped alone -- its rows' layer-0 K/V
 *                       projection; k = floor(t_W / t_d) and T = n_w_total * k;
 *                       in KV_AND_W each weight layer is followed by k dropped
 *                       chunks (the stage's progress is read from the unit
 *                       counts: chunks taken = min(T, all chunks) - N_KV,
 *                       weights taken = n_w_total - N_W; the next unit is a
 *                       weight layer iff chunks taken >= k * weights taken);
 *   MZ_SIZE_RULE_TOTAL  T = the largest n such that dropping the n front-most
 *                       chunks (the last n of the backward-out order, nothing
 *                       else dropped) costs no more recompute time than
 *                       reloading all n_w_total weight layers; in KV_AND_W the
 *                       next chunk is dropped if the recompute total with it
 *                       does not pass the link total, else the next weight
 *                       layer is evicted.
 * Units are taken one at a time, rearmost first, until `bytes` are released:
 *   N_KV > T          KV_ONLY: the next chunk is dropped iff the recompute
 *                     total with it stays below the link total with it
 *                     swapped, else swapped;
 *   N_KV > 0, N_W > 0 KV_AND_W: weight layers and dropped chunks, paired by
 *                     the rule above (paper rule: also with N_W = 0 while
 *                     the weight layers taken cover chunks not yet taken);
 *   N_KV > 0, N_W = 0 the KV_ONLY rule (no weight layer left to pair with);
 *   N_W > 0           W_ONLY: the next weight layer;
 *   otherwise         EXHAUSTED: stop short of `bytes`.
 * Weight layers are evicted as MZ_DROP (reloaded from the library's pinned
 * weight image).  kv_state [n_layers][ceil(n_ctx / chunk_tokens)] and
 * w_state [n_layers] (host) are read as the current states and updated in
 * place.  order (host, NULL or n_layers * (n_chunks + 1) entries) receives
 * the evicted units in eviction order (chunk (l, c) as l * n_chunks + c,
 * weight layer l as n_layers * n_chunks + l), stage (NULL or as many
 * entries) the stage that took each, *n_evicted their count.  info (NULL or
 * 8 doubles): released bytes, T, stage after the call, link total (s),
 * recompute total (s), N_KV, N_W, whether `bytes` was reached (1/0).
 * Errors: EINVAL (sizes, states, non-positive rates, unknown rule). */
mz_status mz_plan_evict_size(const mz_model_cfg *cfg, int32_t n_ctx, const mz_evict_size_request *req,
                             uint8_t *kv_state, uint8_t *w_state, int32_t *order, int32_t *stage,
                             int32_t *n_evicted, double *info);

/* Release at least req->bytes of device memory from ctx's cached context by
 * the policy of mz_plan_evict_size (its kv_codec field is replaced by the
 * context's "kv_codec" option), then mz_evict the planned units in eviction
 * order.  Repeated calls continue from the state the previous ones left.
 * info as in mz_plan_evict_size.  Errors: those of mz_plan_evict_size and
 * mz_evict; ESTATE without a cached context. */
mz_status mz_evict_size(mz_ctx *ctx, const mz_evict_size_request *req, double *info);

/* Bytes of the device GEMM layout of a Q4_0 matrix [n][k] (n padded to 256,
 * k to 64). */
int64_t mz_q4_gemm_packed_bytes(int32_t n, int32_t k);

/* Repack a Q4_0 matrix [n][k] (host, blob row format) into the device GEMM
 * layout (host out, mz_q4_gemm_packed_bytes(n, k) bytes): tiles of 256 rows x
 * 64 columns holding 16-byte code blocks (codes re-ordered for the
 * dequantizer) and then their fp16 scales.  If w_up is not NULL, w and w_up
 * are the gate and up matrices [n][k], each padded to n128 = 128 * ceil(n/128)
 * rows and interleaved in groups of 16 rows (gate group i, then up group i)
 * for the SwiGLU epilogue; out then needs mz_q4_gemm_packed_bytes(2 * n128, k)
 * bytes. */
mz_status mz_q4_gemm_pack(const void *w, const void *w_up, int32_t n, int32_t k, void *out);

/* ---- kernel-level calls (device pointers, enqueue on `stream`) --------- */
/* These run one kernel of the path on caller-owned device buffers; stream is
 * a hipStream_t (NULL = default stream).  They validate shapes and return
 * EINVAL without launching on a mismatch. */

/* Y = X . W^T with X f16 [m][k] row-major (k a multiple of 64) and W packed
 * by mz_q4_gemm_pack (n_pad a multiple of 256; weights dequantized to f16,
 * fp32 accumulation).
 * epilogue 0: y float [m][n_pad] = acc;  1: y float [m][n_pad] += acc;
 * 2: y f16 [m][n_pad/2] = silu(gate) * up (W packed with w_up). */
mz_status mz_q4_gemm(const void *x_f16, int32_t m, int32_t n_pad, int32_t k,
                     const void *w_packed, int32_t epilogue, void *y, void *stream);

/* mz_q4_gemm with persistent workgroups (same arguments, same result bits).
 * The output tiles are cut into 8 contiguous ranges, one per XCD; each
 * workgroup takes tiles of its XCD's range from a counter, then those left
 * in the other ranges, so XCDs that run at a higher clock take more of them.
 * Launches of fewer than 16 rounds of resident workgroups (4096 256-row
 * tiles on 256 compute units) run one workgroup per tile, as mz_q4_gemm.
 * work_queues: device, caller-owned, 16 int32 that are zero before the first
 * call; each call leaves them zero.  Calls that share them must not be in
 * flight at the same time.  EINVAL as mz_q4_gemm, and for a NULL
 * work_queues. */
mz_status mz_q4_gemm_queued(const void *x_f16, int32_t m, int32_t n_pad, int32_t k,
                            const void *w_packed, int32_t epilogue, void *y, int32_t *work_queues,
                            void *stream);

/* Optional parts of a projection launch (mz_q4_gemm_ex), as the restore
 * issues it; a zeroed struct means none of them. */
typedef struct {
  const int32_t *a_rows;     /* device int32 [m]: output row r is computed from X row a_rows[r]
                                (NULL: from X row r) */
  int32_t *work_queues;      /* device, 16 int32 zero on entry and left zero, as in mz_q4_gemm_queued
                                (NULL: one workgroup per tile); epilogues 0-2 only */
  void *workspace;           /* device scratch, not shared with launches in flight: the rows after the
                                last whole 256-row tile run split over K in it (as mz_q4_gemm_split)
                                when their tiles alone would leave most compute units idle (NULL:
                                they run as 64-row tiles); and a product with too few 256-row tiles
                                for the GPU but a long K range runs in it as 256-row tiles split over
                                K (mz_q4_gemm_long_k_splits; NULL: as 64-row tiles over all of K) */
  int64_t workspace_bytes;
  /* rotary epilogues (Sec. 2.1 prefill, rotate-half pairs i, i + head_dim/2 of every head) */
  const int32_t *pos;        /* device int32 [m]: position of output row r */
  const void *rope_cs;       /* device float2 [max(pos) + 1][head_dim / 2]: (cos, sin) of
                                pos * rope_theta^(-2i / head_dim) */
  const int64_t *kv_off;     /* epilogue 5, device int64 [m]: byte offset in slab of row r's key row
                                in its chunk slot, or -1: the row writes nothing */
  void *slab;                /* epilogue 5, device: chunk slots laid out as in mz_attention */
  int32_t head_dim;          /* 32, 64 or 128 */
  int32_t n_valid;           /* epilogue 4: query columns (y row stride); 5: 2 * key columns */
  int32_t chunk_tokens;      /* epilogue 5: tokens per slot, a power of two */
} mz_q4_gemm_args;

/* mz_q4_gemm with the optional parts of mz_q4_gemm_args (args NULL: none),
 * the launch the restore makes for each projection of the prefill that
 * recomputes dropped chunks (paper Sec. 2.1 and 4.2).  Epilogues 0-2 as in
 * mz_q4_gemm; 4: y f16 [m][n_valid] = the rotated queries; 5: columns
 * [0, n_valid/2) are keys, rotated and stored as f16 at slab + kv_off[r],
 * columns [n_valid/2, n_valid) values, stored as f16 into the same slot's
 * V^T half at its position's column (y is not used).  Results equal
 * mz_q4_gemm's bit for bit where no row runs split over K, and to the order
 * of the fp32 sums where one does.  The caller keeps pos, kv_off and a_rows
 * inside their tables and buffers.  Errors: EINVAL for the shapes of
 * mz_q4_gemm, a bad epilogue, missing pointers an epilogue needs, n_valid
 * outside 1..n_pad, head_dim not 32/64/128, chunk_tokens not a power of two. */
mz_status mz_q4_gemm_ex(const void *x_f16, int32_t m, int32_t n_pad, int32_t k, const void *w_packed,
                        int32_t epilogue, const mz_q4_gemm_args *args, void *y, void *stream);

/* One activation row times the packed matrix in a single launch, with any
 * epilogue of mz_q4_gemm_ex: the projections of a decode step and of a
 * restore layer that carries one row (the prefill of Sec. 2.1 and 4.2 at
 * m = 1).  Each workgroup owns a few output columns over the whole K range
 * and applies the epilogue itself, so no workspace and no second kernel are
 * needed.  The row is X row args->a_rows[0] (row 0 without a_rows); with
 * h_norm (device fp32 [.][k]) x_f16 is not read and the row is the RMSNorm
 * of h_norm's row with eps, formed as mz_rmsnorm forms it (the same f16
 * values).  args as in mz_q4_gemm_ex for one output row (pos[0], kv_off[0]);
 * work_queues and workspace must be NULL.  The products of the 4-bit codes
 * with the f16 activations are exact and each block's scale is applied to
 * its fp32 sum, so no weight is rounded to f16 (mz_q4_gemm rounds
 * d * (q - 8) to f16): results agree with mz_q4_gemm's to that rounding and
 * the order of the fp32 sums.  Errors: EINVAL for n_pad not a positive
 * multiple of 256, k not a multiple of 64 or above 16384, the epilogue and
 * pointer errors of mz_q4_gemm_ex, a negative eps, or a workspace. */
mz_status mz_q4_gemv(const void *x_f16, int32_t k, const void *w_packed, int32_t n_pad, int32_t epilogue,
                     const mz_q4_gemm_args *args, const float *h_norm, float eps, void *y, void *stream);

/* Split-K form of mz_q4_gemm for few rows (the short requests of the
 * paper's evaluation, Sec. 6, and every decode step): a grid of 256-column
 * tiles alone leaves most of the GPU idle there.  The k / 64 steps are cut
 * into n_split ranges of ceil((k / 64) / n_split) steps; each range runs as
 * its own workgroups and leaves its fp32 sums in workspace; a second kernel
 * adds the ranges in order and applies the epilogue, so results are
 * deterministic and equal mz_q4_gemm's up to the order of the fp32 sums.
 * workspace: device, caller-owned, at least
 * mz_q4_gemm_split_workspace_bytes(m, n_pad, n_split) bytes, not shared by
 * calls in flight together.  Other arguments and errors as mz_q4_gemm; EINVAL
 * also for n_split outside 1..1024 or a short workspace. */
mz_status mz_q4_gemm_split(const void *x_f16, int32_t m, int32_t n_pad, int32_t k,
                           const void *w_packed, int32_t epilogue, void *y, int32_t n_split,
                           void *workspace, int64_t workspace_bytes, void *stream);

/* Workspace bytes of mz_q4_gemm_split (-1 for invalid arguments). */
int64_t mz_q4_gemm_split_workspace_bytes(int32_t m, int32_t n_pad, int32_t n_split);

/* Size of the fixed device array that holds the partials of
 * mz_q4_gemm_split_noalloc: 32 MiB on each GPU the library runs it on. */
#define MZ_NOALLOC_SCRATCH_BYTES (32 * 1024 * 1024)

/* mz_q4_gemm_split for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, hosts that forbid allocation.  The
 * same kernels and the same result bits as mz_q4_gemm_split with n_split, but
 * the fp32 partials go to a fixed device array of MZ_NOALLOC_SCRATCH_BYTES
 * that the library holds on each GPU it has run this call on, until the
 * process ends; the call allocates nothing.  The array's address on a device
 * is looked up on the first call there, with that device current.  stream
 * (NULL = the default stream) must belong to the current device.  Every call
 * on one GPU shares that GPU's array: calls that overlap on one GPU race
 * (serialize them, e.g. on one stream).  Errors: EINVAL as mz_q4_gemm_split,
 * and when n_split * m * n_pad * 4 bytes exceed MZ_NOALLOC_SCRATCH_BYTES or
 * the stream is on another device (checked before any GPU work); EHIP when no
 * device is usable or the array's address cannot be found. */
mz_status mz_q4_gemm_split_noalloc(const void *x_f16, int32_t m, int32_t n_pad, int32_t k,
                                   const void *w_packed, int32_t epilogue, void *y, int32_t n_split,
                                   void *stream);

/* The split count the restore uses for this shape with workspace_bytes of
 * workspace: about two workgroups per compute unit, at least 4 K steps per
 * split, at most 32 splits; 1 when the tile grid already fills the GPU, or
 * when m >= 1024 and the tiles cover half of its compute units. */
int32_t mz_q4_gemm_auto_splits(int32_t m, int32_t n_pad, int32_t k, int64_t workspace_bytes);

/* The K splits mz_q4_gemm_ex takes with workspace_bytes of workspace when
 * the product's 256-row tiles alone are too few for the GPU while its 64-row
 * tiles fill it: 256-row tiles split into about one round of the compute
 * units, when every split keeps at least 16 K steps of 64 and the fp32
 * partials (splits x m x n_pad x 4 bytes) fit the workspace; 1 otherwise
 * (64-row tiles over the whole K range).  Host only, no GPU work. */
int32_t mz_q4_gemm_long_k_splits(int32_t m, int32_t n_pad, int32_t k, int64_t workspace_bytes);

/* Causal GQA attention (paper Sec. 2.1; read through the chunk table as in
 * Sec. 4.2) of q (f16 [m][n_q_heads][head_dim], rotated) at positions qpos
 * (int32 [m], ascending) over the KV chunks of one layer: chunk c of the
 * layer lives in slot table[c] of slab.  A slot holds K
 * token-major ([chunk_tokens][n_kv_heads * head_dim] f16) followed by V
 * dimension-major ([n_kv_heads * head_dim][chunk_tokens] f16); chunk_tokens is
 * a power of two and a multiple of 8.  Keys 0..qpos[i] are read; table must
 * cover chunk (qpos[m-1] / chunk_tokens) and has n_table entries, at most
 * 8192.  out: f16 [m][n_q_heads * head_dim]. */
mz_status mz_attention(const void *q_f16, const int32_t *qpos, int32_t m, const void *slab,
                       const int32_t *table, int32_t n_table, int32_t chunk_tokens,
                       int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim, void *out_f16,
                       void *stream);

/* mz_attention with persistent workgroups that take the query tiles from
 * per-KV-head work queues (same arguments, same result bits).  Each XCD first
 * serves the queue of its own KV head, heaviest tiles first, then takes the
 * lightest tiles left in the others, so XCDs that run at a higher clock take
 * more of the work.  work_queues: device, caller-owned, 16 int32 that are
 * zero before the first call; each call leaves them zero.  Calls that share
 * them must not be in flight at the same time.  Where n_kv_heads does not
 * divide 8 or chunk_tokens < 64 this runs as mz_attention.  EINVAL as
 * mz_attention, and for a NULL work_queues. */
mz_status mz_attention_queued(const void *q_f16, const int32_t *qpos, int32_t m, const void *slab,
                              const int32_t *table, int32_t n_table, int32_t chunk_tokens,
                              int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim, void *out_f16,
                              int32_t *work_queues, void *stream);

/* Split-key form of mz_attention for few query rows against a long context
 * (the paper's short requests, Sec. 6; the attention of its custom kernel,
 * Sec. 4.2, is one pass over the chunks, which leaves most of the GPU idle
 * when there are few queries).  The keys 0..max_pos are cut into n_split
 * ranges of whole 64-key tiles, ceil((max_pos / 64 + 1) / n_split) tiles
 * each; every range runs as its own workgroups and leaves, per query row and
 * head, its output normalised by its own softmax sum (f16) with that sum and
 * the running max (fp32) in workspace; a second kernel merges the ranges
 * with weights 2^(max_s - max) * sum_s.  The result equals mz_attention's to
 * the f16 rounding of the partial outputs.  max_pos (host value) must be >=
 * qpos[m-1], and table must cover chunk max_pos / chunk_tokens.  workspace:
 * device, caller-owned, at least mz_attention_split_workspace_bytes(m,
 * n_q_heads, head_dim, n_split) bytes; it must not be shared by calls in
 * flight at the same time.  Other arguments and errors as mz_attention;
 * EINVAL also for n_split outside 1..64 or a short workspace. */
mz_status mz_attention_split(const void *q_f16, const int32_t *qpos, int32_t m, int32_t max_pos,
                             const void *slab, const int32_t *table, int32_t n_table,
                             int32_t chunk_tokens, int32_t n_q_heads, int32_t n_kv_heads,
                             int32_t head_dim, int32_t n_split, void *workspace,
                             int64_t workspace_bytes, void *out_f16, void *stream);

/* Workspace bytes of mz_attention_split (-1 for invalid arguments). */
int64_t mz_attention_split_workspace_bytes(int32_t m, int32_t n_q_heads, int32_t head_dim,
                                           int32_t n_split);

/* The split count the restore uses for m query rows up to max_pos with
 * workspace_bytes of workspace: enough workgroups for two per compute unit
 * (one where the m rows make at most 16 (row, query head) columns per KV
 * head, the few-column kernel), at least 4 key tiles per split, at most 64
 * splits; 1 when the unsplit kernel already fills the GPU. */
int32_t mz_attention_auto_splits(int32_t m, int32_t max_pos, int32_t n_q_heads, int32_t n_kv_heads,
                                 int32_t head_dim, int64_t workspace_bytes);

/* x = h / sqrt(mean(h^2) + eps) per row: h float [m][d] -> x f16 [m][d]. */
mz_status mz_rmsnorm(const void *h_f32, int32_t m, int32_t d, float eps, void *x_f16,
                     void *stream);

/* 8-bit group-wise codec of the swap path (paper Sec. 5: 8-bit quantization
 * as the default KV codec).  On n_halves IEEE halves (a positive multiple of
 * 64), in groups of 64 consecutive values: mn, mx = min, max;
 * d = half(fp32(mx - mn) / 255); q = d == 0 ? 0 : clamp(rint(fp32(x - mn) /
 * fp32(d)), 0, 255) (correctly rounded division, ties to even);
 * x^ = half(fp32(q) * fp32(d) + fp32(mn)).  Compressed layout (device, caller
 * owned): n_halves code bytes, then (mn, d) as two halves per group, i.e.
 * n_halves + n_halves / 16 bytes.  Enqueued on stream. */
mz_status mz_kv_compress(const void *src_f16, int64_t n_halves, void *out, void *stream);
mz_status mz_kv_decompress(const void *in, int64_t n_halves, void *dst_f16, void *stream);

/* Ceilings this GPU actually sustains, measured on the spot (not part of the
 * restore path; for stating measured rates against them): f16 MFMA
 * throughput with operand bits that keep changing as real data does, a plain
 * 1 GiB device copy (bytes read + written), and 1 GiB pinned host -> device
 * and device -> host copies.  Two more MFMA figures price an exact-integer
 * weight operand: "mfma_f16_codes_tflops" with one operand holding exact
 * 4-bit codes q - 8, and "mfma_f16_block_scaled_tflops" with, in addition,
 * each 32-deep product summed into a zero accumulator and scaled into the
 * running sum by four fp32 FMAs (a Q4_0 block scale applied after the
 * product).  Writes JSON
 * {"mfma_f16_tflops", "mfma_f16_codes_tflops", "mfma_f16_block_scaled_tflops",
 *  "hbm_copy_gbps", "h2d_pinned_gbps", "d2h_pinned_gbps"}
 * into json_out (cap bytes, NUL-terminated).  Allocates and frees about
 * 2 GiB of device memory and 1 GiB of pinned host memory; takes about
 * two seconds.  Errors: MZ_EINVAL (buffer), MZ_ENOMEM / MZ_EHIP (device). */
mz_status mz_probe_ceilings(int32_t device, char *json_out, size_t cap);

#ifdef __cplusplus
}
#endif

#endif /* MZ_H */
