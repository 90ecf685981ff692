/*
 * acache.h — C ABI of the selective affix-KV recompute path for MI355X (gfx950).
 *
 * The operation is ACache's ("Affix Cache for Diffusion Large Language
 * Models"): a shared affix keeps one precomputed KV cache; each request picks
 * Anchor Tokens once by a probe that scores affix tokens with the attention
 * they receive from masked generation queries (Section 3.2, Eq. 4-6); at
 * every recomputation point only the anchors and the request-specific
 * positions are recomputed, while the other affix tokens keep the shared
 * cache (Section 3.3).  Recomputed KV goes to request-private slots through a
 * write-side map, and attention reads the full logical context through a
 * read-slot map (Section 4.1, Appendix C.1).
 *
 * Conventions for every call:
 *  - Pointers are DEVICE pointers unless marked [host].  Host arrays are read
 *    during the call only.
 *  - Ownership: the caller owns every buffer.  The library allocates and
 *    frees no device memory and never synchronises; work is enqueued on
 *    `stream` and the call returns.  Buffers must stay alive until the
 *    stream has passed the work.  The only global state is the opt-in
 *    measurement hook (acache_time_kernel).
 *  - Errors: host-checkable faults (NULL pointers, sizes, alignment,
 *    unsupported shapes, a workspace that is too small) return a non-zero
 *    status and enqueue nothing.  A failed launch returns ACACHE_ERR_DEVICE.
 *  - Device-resident indices (slots, rows, anchors) are checked on the
 *    device against the sizes passed here: an out-of-range index is skipped
 *    (its read yields zeros, its write is dropped), never dereferenced.
 *  - Element types: ACACHE_BF16 is bfloat16 storage with fp32 accumulation;
 *    ACACHE_F32 is fp32 throughout.  Weights, activations and KV pools share
 *    the `dims->dtype` storage type; scores and log-sum-exp are fp32.
 *  - Row-major layouts.  A KV pool is [n_slots, pool_ld] elements, one pool
 *    per layer for K and one for V; the row of a slot holds H_kv heads of
 *    head_dim elements (K after rotation).  Leading dimensions are in
 *    elements unless named *_bytes.  The kernels address a pool with 32-bit
 *    element offsets: acache_score, acache_attention and
 *    acache_layer_recompute return ACACHE_ERR_UNSUPPORTED unless
 *    n_slots * pool_ld < 2^31.
 *  - The fused block is the LLaDA / Dream family's: RMSNorm, Q/K/V
 *    projections (no bias), rotary embedding on half-split pairs at the
 *    row's position, bidirectional attention with grouped KV heads, output
 *    projection + residual, RMSNorm, SwiGLU MLP + residual.
 */
#ifndef ACACHE_H
#define ACACHE_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  ACACHE_OK = 0,
  ACACHE_ERR_NULL = 1,        /* a required pointer is NULL */
  ACACHE_ERR_SHAPE = 2,       /* sizes are negative, inconsistent or out of range */
  ACACHE_ERR_ALIGN = 3,       /* a pointer or leading dimension is not 16-byte aligned */
  ACACHE_ERR_UNSUPPORTED = 4, /* valid, but outside the shapes the kernels implement */
  ACACHE_ERR_WORKSPACE = 5,   /* workspace NULL or smaller than acache_workspace_size() */
  ACACHE_ERR_DEVICE = 6,      /* a HIP launch or call failed */
  ACACHE_ERR_SPACE = 7        /* a block pool has fewer free blocks than asked for */
} acache_status;

typedef enum { ACACHE_F32 = 0, ACACHE_BF16 = 1 } acache_dtype;

/* Normalisation of the Eq. 4 softmax.  AFFIX: over the affix keys only, as
 * Eq. 4 is written.  FULL: the model's softmax over every key of the
 * request, read through the per-row log-sum-exp the attention exports. */
typedef enum { ACACHE_NORM_AFFIX = 0, ACACHE_NORM_FULL = 1 } acache_norm;

typedef struct {
  int32_t d_model;    /* hidden size d */
  int32_t n_heads;    /* query heads H */
  int32_t n_kv_heads; /* KV heads H_kv; H % H_kv == 0 (head h reads KV head h / (H / H_kv)) */
  int32_t head_dim;   /* d_h */
  int32_t d_ff;       /* SwiGLU width F */
  float rms_eps;      /* RMSNorm epsilon */
  float rope_base;    /* rotary base: theta_i = base^(-2i / d_h) */
  acache_dtype dtype;
} acache_dims;

/* One layer's weights, [out_features, in_features] row-major, dims->dtype. */
typedef struct {
  const void* attn_norm; /* [d]                      RMSNorm gain before attention */
  const void* w_qkv;     /* [(H + 2 H_kv) d_h, d]    rows: Q heads, K heads, V heads */
  const void* w_o;       /* [d, H d_h] */
  const void* mlp_norm;  /* [d]                      RMSNorm gain before the MLP */
  const void* w_gate_up; /* [2 F, d]                 rows: F gate rows, then F up rows */
  const void* w_down;    /* [d, F] */
} acache_layer_weights;

/* A ragged batch.  Request b owns rows [cu_rows[b], cu_rows[b+1]) of the
 * row-indexed buffers and reads its logical keys through
 * read_slots[cu_keys[b] .. cu_keys[b+1]).  batch <= 64. */
typedef struct {
  int32_t batch;
  const int32_t* cu_rows; /* [host] batch + 1, nondecreasing, cu_rows[0] == 0 */
  const int32_t* cu_keys; /* [host] batch + 1, nondecreasing, cu_keys[0] == 0 */
} acache_ragged;

/* Probe scoring inside acache_layer_recompute (Section 3.2, Eq. 4-5). */
typedef struct {
  const int32_t* q_rows;      /* [cu_q[batch]] rows (of this layer's rows) of the masked queries */
  const int32_t* cu_q;        /* [host] batch + 1: request b's masked rows are q_rows[cu_q[b] ..) */
  const int32_t* affix_slots; /* [affix_len] pool slots of the affix keys, affix-local order */
  int32_t affix_len;          /* L */
  acache_norm norm;
  float* scores;              /* [batch, L] fp32, accumulated (+=) */
  int32_t init;               /* nonzero: scores = this layer's sum, not read first (a probe's first
                                 layer, so the caller need not clear scores).  Applies only to a call
                                 that scores (L > 0 and some masked rows); otherwise scores is left
                                 unchanged, as with init == 0 */
  int32_t affix_keys_known;   /* acache_layer_recompute only; nonzero: every request's read slots hold
                                 the affix keys in affix-local order from key index affix_key_begin,
                                 read_slots[cu_keys[b] + affix_key_begin + j] == affix_slots[j] for
                                 j < L.  Under ACACHE_NORM_AFFIX on the bf16 path the attention pass
                                 then also takes each row's log-sum-exp over those keys and the score
                                 uses it instead of its own pass over the affix keys (when
                                 affix_key_begin is 0 and L is a multiple of 64; otherwise the score
                                 makes that pass itself).  Zero: no such promise (any caller that
                                 leaves the field zeroed) */
  int32_t affix_key_begin;    /* with affix_keys_known: key index of the first affix key, >= 0, the same
                                 in every request; each request has at least affix_key_begin + L keys,
                                 or the promise is ignored */
} acache_score_args;

/* Logical layout shared by every request of a batch, and its slot plan. */
typedef struct {
  int32_t seq_len;        /* S: logical positions per request, 0 .. S-1 */
  int32_t affix_begin;    /* first position of the shared affix span */
  int32_t affix_len;      /* L */
  int32_t mask_begin;     /* first position of the masked generation span M_T */
  int32_t mask_len;       /* G */
  int32_t shared_base;    /* pool slot of affix-local index 0 (shared region) */
  int32_t private_base;   /* first private slot */
  int32_t private_stride; /* request b's private slots start at private_base + b * private_stride */
  int32_t key_order;      /* order of a request's keys in read_slots: 0, logical positions 0 .. S-1;
                             1, the L affix positions first (affix-local order), then the others in
                             logical order.  Attention over a request's keys does not depend on their
                             order; the probe reads the affix first so that its attention pass can
                             take the affix log-sum-exp of Eq. 4 (acache_score_args) */
} acache_layout;

/* ---------------------------------------------------------------------------
 * acache_score — Eq. 4-5 of Section 3.2 for one layer: for every request b,
 * masked query row k (q_rows[cu_q[b] ..)), head h and affix key j,
 *   a = softmax over the affix keys of q_k . K_j / sqrt(d_h)   (AFFIX), or
 *   a = exp(q_k . K_j / sqrt(d_h) - row_lse[k, h])              (FULL),
 * and scores[b, j] += sum over h and k of a.  Keys are k_pool[affix_slots[j]],
 * KV head h / (H / H_kv).  The sum is taken in a fixed order (no float
 * atomics): identical inputs give identical bits.
 *   q        [rows, q_ld] post-rotation queries, head h at columns h*d_h
 *   row_lse  [rows, H] natural-log log-sum-exp of the scaled logits over all
 *            of the row's keys (as acache_attention exports); required for
 *            FULL, must be NULL for AFFIX
 *   ws       workspace of at least acache_workspace_size() bytes
 * Requires head_dim == 128 (bf16) or head_dim <= 128 (f32); L <= 65536.
 * L == 0 or no masked rows: no-op. */
acache_status acache_score(const acache_dims* dims, int32_t batch, const void* q, int64_t q_ld,
                           int64_t q_n_rows, const int32_t* q_rows, const int32_t* cu_q,
                           const void* k_pool, int64_t pool_ld, int64_t n_slots,
                           const int32_t* affix_slots, int32_t affix_len, const float* row_lse,
                           acache_norm norm, float* scores, void* ws, size_t ws_bytes,
                           hipStream_t stream);

/* ---------------------------------------------------------------------------
 * acache_score_noalloc — acache_score without a workspace, for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc).  Same arguments, kernels and
 * results as acache_score, bit for bit.  Its scratch (the per-row
 * log-sum-exp and per-head column sums) is a fixed array in the library's
 * device memory, one per GPU, held until the process ends; the call neither
 * allocates nor frees.  Limit: cu_q[batch] * H * 4 + batch * H * affix_len * 4
 * bytes (each rounded up to 256) must not exceed
 * acache_score_noalloc_max_bytes() (64 MiB), else ACACHE_ERR_WORKSPACE with
 * nothing enqueued.  Every call on one GPU uses that GPU's one scratch:
 * calls that overlap on one GPU (other streams, other threads) race; calls
 * ordered on one stream do not.  The first call on a device resolves the
 * scratch address on that device (the device must be current). */
acache_status acache_score_noalloc(const acache_dims* dims, int32_t batch, const void* q, int64_t q_ld,
                                   int64_t q_n_rows, const int32_t* q_rows, const int32_t* cu_q,
                                   const void* k_pool, int64_t pool_ld, int64_t n_slots,
                                   const int32_t* affix_slots, int32_t affix_len, const float* row_lse,
                                   acache_norm norm, float* scores, hipStream_t stream);
size_t acache_score_noalloc_max_bytes(void);

/* ---------------------------------------------------------------------------
 * acache_anchor_count — the K of Eq. 6 for anchor ratio `ratio` over an affix
 * of affix_len tokens: the integer nearest to ratio * affix_len, a half
 * rounded up (the paper states no rounding; 0.2 of 128 tokens is 26), within
 * [0, affix_len].  Host-side arithmetic, no device work.  Returns -1 if
 * ratio is outside [0, 1] (or NaN) or affix_len < 0. */
int32_t acache_anchor_count(double ratio, int32_t affix_len);

/* ---------------------------------------------------------------------------
 * acache_topk — Eq. 6: per request b, the k indices j of the largest
 * scores[b, j], written ascending to idx_out[b, 0..k).  Ties go to the lowest
 * index; -0 equals +0; NaN ranks below every other value (-inf included).
 * Exact: the selection compares order-preserving integer keys of the fp32
 * bits.  0 <= k <= L <= 16384; k == 0 is a no-op. */
acache_status acache_topk(const float* scores, int32_t batch, int32_t L, int32_t k,
                          int32_t* idx_out, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * acache_gather_rows — queries are formed only for recomputed positions
 * (Section 4.3): dst row i = src row r, r = remap ? remap[idx[i]] : idx[i],
 * for i < n.  Rows are row_bytes long (multiple of 16); src rows
 * 0 .. src_rows-1 exist; remap has remap_len entries.  Pointers and
 * leading dimensions 16-byte aligned.  n == 0: no-op. */
acache_status acache_gather_rows(const void* src, int64_t src_ld_bytes, int64_t src_rows,
                                 const int32_t* idx, const int32_t* remap, int64_t remap_len,
                                 int32_t n, int32_t row_bytes, void* dst, int64_t dst_ld_bytes,
                                 hipStream_t stream);

/* ---------------------------------------------------------------------------
 * acache_kv_scatter — the store half of store-then-attend (Appendix C.1):
 * k_pool[dst_slots[i]] = k_src row i and v_pool[dst_slots[i]] = v_src row i,
 * row_elems elements each (multiple of 8), for i < n.  Sources are
 * [n, src_ld]; pools [n_slots, pool_ld].  n == 0: no-op. */
acache_status acache_kv_scatter(const void* k_src, const void* v_src, int64_t src_ld, int32_t n,
                                const int32_t* dst_slots, void* k_pool, void* v_pool,
                                int64_t pool_ld, int64_t n_slots, int32_t row_elems,
                                acache_dtype dtype, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * acache_build_maps — the write-side recomputation map and the read-slot
 * map of Section 4.1, built on the device from the anchor lists.  For
 * request b the recomputed positions are every non-affix position plus
 * affix_begin + anchors[b, i]; taken in ascending order they are rows
 * b*R .. b*R + R-1 (R = k + S - L) and get private slots
 * private_base + b*private_stride + (rank).  Outputs:
 *   row_pos     [B*R]  logical position of each recomputed row
 *   row_src     [B*R]  b*S + position (index into per-position inputs)
 *   write_slots [B*R]  private slot of each recomputed row
 *   read_slots  [B*S]  slot each key is read from, keys in the layout's key_order
 *                      (key_order 0: key p is logical position p): its private slot
 *                      if recomputed, else shared_base + (p - affix_begin)
 *   q_rows      [B*G]  (nullable) row of each masked position
 * anchors [B, k] affix-local indices, ascending per request (NULL iff k == 0).
 * k == 0 gives the probe / direct-reuse maps, k == L the full-recompute maps.
 * Requires private_stride >= R. */
acache_status acache_build_maps(const acache_layout* layout, int32_t batch,
                                const int32_t* anchors, int32_t k, int32_t* row_pos,
                                int32_t* row_src, int32_t* write_slots, int32_t* read_slots,
                                int32_t* q_rows, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Block-granular KV slots (Section 4.1: the shared prefix cache sits in
 * reserved shared blocks, and each request's anchors and request-specific
 * positions in private blocks; peak KV use is then counted in whole blocks,
 * the granularity behind the batch-1 overhead discussed with Table 4).
 *
 * A paged slot plan: slots come in blocks of block_size consecutive slots,
 * block id i covering slots i*block_size .. i*block_size + block_size-1.
 *   affix-local index j      -> shared_blocks[j / bs] * bs + j % bs
 *   request b's rank-i row   -> private_blocks[b * blocks_per_request + i / bs] * bs + i % bs
 * (bs = block_size).  shared_blocks [ceil(L / bs)] and private_blocks
 * [batch * blocks_per_request] are DEVICE arrays of block ids >= 0; a slot
 * that would not fit in int32 is written as -1, which every consumer skips.
 */
typedef struct {
  int32_t block_size;
  int32_t blocks_per_request;
  const int32_t* shared_blocks;
  const int32_t* private_blocks;
} acache_paging;

/* acache_build_maps_paged — acache_build_maps with the slots of a paged
 * plan in place of shared_base / private_base / private_stride (which it
 * ignores): the same rows, positions and order.  Requires block_size >= 1
 * and blocks_per_request * block_size >= R. */
acache_status acache_build_maps_paged(const acache_layout* layout, const acache_paging* paging,
                                      int32_t batch, const int32_t* anchors, int32_t k, int32_t* row_pos,
                                      int32_t* row_src, int32_t* write_slots, int32_t* read_slots,
                                      int32_t* q_rows, hipStream_t stream);

/* acache_block_pool — a host-side allocator of block ids 0 .. capacity-1
 * (no device memory: the caller sizes the KV pools to capacity blocks).
 * alloc writes n ids to ids [host] — the lowest free ones, ascending — or
 * returns ACACHE_ERR_SPACE and allocates nothing; free returns n allocated
 * ids (ACACHE_ERR_SHAPE, and nothing freed, for an id out of range, not
 * allocated, or listed twice).  stats reports capacity, blocks in use and
 * the peak in use since creation or reset_peak (any output may be NULL).
 * A pool is not thread-safe. */
typedef struct acache_block_pool acache_block_pool;
acache_status acache_block_pool_create(int32_t capacity, acache_block_pool** pool);
acache_status acache_block_pool_destroy(acache_block_pool* pool);
acache_status acache_block_pool_alloc(acache_block_pool* pool, int32_t n, int32_t* ids);
acache_status acache_block_pool_free(acache_block_pool* pool, int32_t n, const int32_t* ids);
acache_status acache_block_pool_stats(const acache_block_pool* pool, int32_t* capacity, int32_t* in_use,
                                      int32_t* peak);
acache_status acache_block_pool_reset_peak(acache_block_pool* pool);

/* ---------------------------------------------------------------------------
 * acache_attention — read-slot attention (Appendix C.1): for request b,
 * head h and each query row r in [cu_rows[b], cu_rows[b+1]),
 *   out[r, h] = softmax_j(q[r, h] . K_j / sqrt(d_h)) V_j
 * over the request's logical keys j, K_j = k_pool[read_slots[cu_keys[b] + j]]
 * (KV head h / (H / H_kv)), bidirectional, no mask.  q and out are
 * [rows, H*d_h]; lse (nullable) [rows, H] receives the natural-log
 * log-sum-exp of the scaled logits.  A request with rows must have keys. */
acache_status acache_attention(const acache_dims* dims, const acache_ragged* rg, const void* q,
                               const int32_t* read_slots, const void* k_pool, const void* v_pool,
                               int64_t pool_ld, int64_t n_slots, void* out, float* lse,
                               hipStream_t stream);

/* ---------------------------------------------------------------------------
 * acache_layer_recompute — one block over the recomputed rows of a ragged
 * batch (Sections 3.3 and 4.3): with y = RMSNorm(x) the rows' Q, K, V are
 * projected, rotated at pos[r], the fresh K/V stored at write_slots[r], and
 * then attention reads every logical key through read_slots (store, then
 * attend).  x is updated in place:
 *   x += Attn(...) W_o^T;  x += (SiLU(y2 Wg^T) * (y2 Wu^T)) W_down^T,  y2 = RMSNorm(x).
 * With `score` set (the probe of Section 3.2), this layer's Eq. 4-5
 * contribution is added to score->scores from the masked rows' queries
 * against the affix keys, as acache_score does.
 *   x           [rows, d] in/out, rows = cu_rows[batch]
 *   pos         [rows] logical position of each row (rotation angle)
 *   write_slots [rows] pool slot receiving each row's K and V
 *   read_slots  [cu_keys[batch]] slots of each request's logical keys
 *   pools       [n_slots, pool_ld], pool_ld >= H_kv * d_h
 *   ws          at least acache_workspace_size(dims, rows, batch, L) bytes
 * bf16 requires head_dim == 128, d_model % 256 == 0, (H*d_h) % 256 == 0,
 * (H_kv*d_h) % 128 == 0, d_ff % 128 == 0; f32 requires head_dim % 2 == 0,
 * head_dim <= 128.  The projections use 32-bit element offsets: rows times
 * max(d, H*d_h, d_ff) and every weight matrix must stay below 2^31 elements
 * (ACACHE_ERR_UNSUPPORTED otherwise; split a larger batch into calls). */
acache_status acache_layer_recompute(const acache_dims* dims, const acache_layer_weights* w,
                                     const acache_ragged* rg, void* x, const int32_t* pos,
                                     const int32_t* write_slots, const int32_t* read_slots,
                                     void* k_pool, void* v_pool, int64_t pool_ld, int64_t n_slots,
                                     const acache_score_args* score, void* ws, size_t ws_bytes,
                                     hipStream_t stream);

/* ---------------------------------------------------------------------------
 * acache_layer_score — the probe's last layer (Section 3.2, Eq. 4-5) reduced
 * to what its score reads.  After the last probe layer nothing consumes the
 * probe rows' hidden states (the refresh recomputes every row from its
 * layer-0 input), so only this layer's Eq. 4 weights matter: with
 * y = RMSNorm(x), the masked rows' queries y W_q^T rotated at pos, against
 * the affix keys, added into score->scores exactly as acache_layer_recompute
 * with the same score arguments does (equal up to fp32 summation order in
 * the query projection).
 *   ACACHE_NORM_AFFIX: only the masked rows (score->q_rows) are normalised
 *     and projected, to queries only; the pools are not written.
 *   ACACHE_NORM_FULL: the normaliser is each masked row's LSE over all of
 *     its request's keys, so every row's Q, K and V are projected, K and V
 *     stored at write_slots, and the attention runs over read_slots (its
 *     output is discarded).
 * x [rows, d] is read only.  score is required.  write_slots, read_slots
 * and v_pool may be NULL under ACACHE_NORM_AFFIX.  The weights read are
 * attn_norm and w_qkv (its first H*d_h rows under AFFIX); the others may be
 * NULL.  Other arguments, layouts, the workspace and the errors are those
 * of acache_layer_recompute; bf16 under AFFIX also needs d_ff >= d_model.
 * No masked rows or L == 0: no-op. */
acache_status acache_layer_score(const acache_dims* dims, const acache_layer_weights* w, const acache_ragged* rg,
                                 const void* x, const int32_t* pos, const int32_t* write_slots,
                                 const int32_t* read_slots, void* k_pool, void* v_pool, int64_t pool_ld,
                                 int64_t n_slots, const acache_score_args* score, void* ws, size_t ws_bytes,
                                 hipStream_t stream);

/* ---------------------------------------------------------------------------
 * acache_kv_deviation — the score of the CacheBlend-style selector the paper
 * compares against (appendix, "CacheBlend-Style Anchor Selection"): each
 * affix token's KV deviation between the shared affix-only cache and the
 * request's full-prompt cache,
 *   scores[b, j] = sum over the row's H_kv * d_h elements of
 *                  (K[f] - K[s])^2 + (V[f] - V[s])^2,
 * f = fresh_slots[b * fresh_ld + j] (the request's full-prompt K/V of affix
 * token j at the selection layer), s = stale_slots[j] (the shared cache),
 * accumulated in fp32 in a fixed order (scores are overwritten).  A row with
 * a slot outside [0, n_slots) scores 0.  Pools [n_slots, pool_ld] of
 * dims->dtype, 16-byte aligned.  The anchors are then acache_topk of the
 * scores (Eq. 6's rule).  batch == 0 or affix_len == 0: no-op. */
acache_status acache_kv_deviation(const acache_dims* dims, int32_t batch, int32_t affix_len, const void* k_pool,
                                  const void* v_pool, int64_t pool_ld, int64_t n_slots, const int32_t* fresh_slots,
                                  int64_t fresh_ld, const int32_t* stale_slots, float* scores, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * acache_rerotate_k — reuse of a cached span at shifted positions (the
 * runtime piece Section 4 and the Limitations leave to future work: the
 * cache is stored after rotation).  Rotations compose, so the K a row would
 * have at position p + delta is its cached K (position p) turned by delta:
 * for every row i < n, k_dst[dst_slots[i]] = rotate(k_src[src_slots[i]],
 * delta[i]), each half-split pair (j, j + d_h/2) of every KV head by
 * delta[i] * theta_j, theta_j = base^(-2j/d_h), the angle reduced in fp64.
 * V is position-free and is not touched.  Pools [n_slots, pool_ld] of
 * dims->dtype, one row = H_kv heads x head_dim; src and dst may be the same
 * pool and the same slots (in place).  Rows whose slots fall outside
 * [0, n_slots) are skipped.  n == 0: no-op. */
acache_status acache_rerotate_k(const acache_dims* dims, const void* k_src, const int32_t* src_slots, void* k_dst,
                                const int32_t* dst_slots, const int32_t* delta, int32_t n, int64_t pool_ld,
                                int64_t n_slots, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * acache_layer_decode — one block of a block-decoding step (Section 4.3:
 * queries for the current block only; Appendix C.1: store, then attend over
 * the read-slot view), computed as acache_layer_recompute would for `batch`
 * requests of rows_per_request rows each (row i of request b is row
 * b * rows_per_request + i of x, pos, write_slots), with request b's logical
 * keys given as two sets instead of one read-slot list:
 *   - the shared affix: slot affix_slots[j] for every affix-local index
 *     j < affix_len that is not one of anchors[b, 0 .. k) (the positions a
 *     refresh recomputed are read from private slots);
 *   - its private keys: private_slots[b * private_len .. + private_len), the
 *     slots of the request's recomputed rows (anchors and request-specific
 *     positions; the block's own rows are among them).
 * The queries of all requests are taken together against the shared affix
 * keys, so each affix K/V tile is read once per 128 queries rather than once
 * per request; the request's private keys follow, and the two softmax
 * partials are merged.  The result equals acache_layer_recompute over the
 * same view up to fp32 summation order.  bf16 only (ACACHE_ERR_UNSUPPORTED
 * otherwise); batch <= 64, affix_len <= 65536.  ws: at least
 * acache_workspace_size(dims, batch * rows_per_request, batch, affix_len)
 * bytes. */
acache_status acache_layer_decode(const acache_dims* dims, const acache_layer_weights* w, int32_t batch,
                                  int32_t rows_per_request, void* x, const int32_t* pos, const int32_t* write_slots,
                                  const int32_t* affix_slots, int32_t affix_len, const int32_t* anchors, int32_t k,
                                  const int32_t* private_slots, int32_t private_len, void* k_pool, void* v_pool,
                                  int64_t pool_ld, int64_t n_slots, void* ws, size_t ws_bytes, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * acache_argmax_commit — the commit half of the predict-then-commit loop
 * (Section 3.1; the online loop of Section 4.3), in its greedy form: for
 * every row i < rows, out[i] = the index of the largest of x[i, 0 .. n),
 * comparing values as numbers with -0 == +0 and NaN below everything, the
 * lowest index among equal values.  conf (nullable, fp32 [rows]) receives
 * the row's confidence, the softmax probability of its largest value,
 * 1 / sum_j exp(x_j - max) over the values that are not NaN or -inf (equal
 * maxima, +inf included, share the mass equally; 0 for a row with none).  With commit_pos (nullable) the index is also written to
 * ids[commit_pos[i]]; positions outside [0, ids_len) are skipped.
 * x [rows, ld] of `dtype` (logits).  rows == 0: no-op; n == 0 with
 * rows > 0: ACACHE_ERR_SHAPE. */
acache_status acache_argmax_commit(acache_dtype dtype, const void* x, int64_t ld, int32_t rows, int32_t n,
                                   int32_t* out, float* conf, const int32_t* commit_pos, int32_t* ids,
                                   int64_t ids_len, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * acache_threshold_commit — one decode step's commit in the block-wise loop
 * (Section 3.1; Section 4.3: during block decoding queries are formed for
 * the current block only; Section 5 commits by a confidence threshold).  For
 * each request b, over its rows r = b * block .. b * block + block - 1 (pick
 * and conf from acache_argmax_commit of the block's logits): every row with
 * committed[r] == 0 and conf[r] >= tau is committed; if none is, the single
 * uncommitted row with the highest conf (the lowest r among equals; NaN
 * lowest).  Committing sets committed[r] = 1 and ids[commit_pos[r]] =
 * pick[r] (skipped outside [0, ids_len)).  count[b] = rows committed by this
 * call (0 once the block is done).  batch == 0: no-op. */
acache_status acache_threshold_commit(int32_t batch, int32_t block, const int32_t* pick, const float* conf, float tau,
                                      int32_t* committed, const int32_t* commit_pos, int32_t* ids, int64_t ids_len,
                                      int32_t* count, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Building blocks of acache_layer_recompute, exported so each can be checked
 * on its own.
 *
 * acache_rmsnorm: y[r] = x[r] / sqrt(mean(x[r]^2) + eps) * g, rows x [rows, d].
 * acache_linear:  c[m, n] = sum_k a[m, k] w[n, k] (+ c[m, n] when accumulate),
 *                 a [M, K], w [N, K], c [M, N], dims->dtype storage, fp32
 *                 accumulation.  bf16 requires K % 64 == 0, N % 256 == 0.
 *                 ws is optional: with a 16-byte aligned bf16 workspace of
 *                 acache_workspace_size(dims, M, 1, 0) bytes or more, row
 *                 counts that leave CUs idle in the last round of tiles are
 *                 balanced by splitting K across workgroups (fp32 partials,
 *                 summed in a fixed order); without it every tile runs whole.
 *                 The two schedules agree up to fp32 summation order.
 *                 M * K and N * K must be below 2^31 (32-bit offsets). */
acache_status acache_rmsnorm(const acache_dims* dims, const void* x, const void* g, void* y,
                             int32_t rows, hipStream_t stream);
acache_status acache_linear(const acache_dims* dims, const void* a, const void* w, void* c,
                            int32_t M, int32_t N, int32_t K, int32_t accumulate,
                            void* ws, size_t ws_bytes, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Measurement hook (benchmarks only).  While armed for kernel `kernel`,
 * every launch of that kernel by any entry point records starts[i] before
 * and stops[i] after it on the launch stream, i = *count, *count + 1, ...,
 * up to `capacity` records; the caller reads the durations with
 * hipEventElapsedTime.  The events are the caller's (hipEventCreate).
 * kernel == ACACHE_K_NONE disarms.  This is the library's only mutable
 * state: arming is not thread-safe and applies to all streams. */
typedef enum {
  ACACHE_K_NONE = -1,
  ACACHE_K_GEMM_QKV = 0,     /* Q/K/V projection + rotary + K/V store */
  ACACHE_K_GEMM_O = 1,       /* output projection (split-K partials) */
  ACACHE_K_GEMM_GATE_UP = 2, /* gate/up projection + SwiGLU */
  ACACHE_K_GEMM_DOWN = 3,    /* down projection (split-K partials) */
  ACACHE_K_ATTENTION = 4,    /* read-slot attention */
  ACACHE_K_SCORE_LSE = 5,    /* probe: affix-only log-sum-exp (fp32 path; bf16 does it in SCORE_COLSUM) */
  ACACHE_K_SCORE_COLSUM = 6, /* probe: per-head column sums (bf16: with the log-sum-exp sweep) */
  ACACHE_K_SCORE_REDUCE = 7, /* probe: fixed-order head reduction */
  ACACHE_K_RMSNORM = 8,      /* RMSNorm before attention */
  ACACHE_K_RESIDUAL = 9,     /* split-K reduction + residual (+ RMSNorm) */
  ACACHE_K_TOPK = 10,
  ACACHE_K_GATHER = 11,
  ACACHE_K_MAPS = 12,
  ACACHE_K_SCATTER = 13,
  ACACHE_K_ARGMAX = 14,
  ACACHE_K_COUNT = 15
} acache_kernel_id;
acache_status acache_time_kernel(int32_t kernel, hipEvent_t* starts, hipEvent_t* stops,
                                 int32_t capacity, int32_t* count);

/* The K splits acache_layer_recompute uses for `rows` rows: of the output
 * projection (*o_splits) and of the down projection (*down_splits).  One
 * split: the projection adds itself to the residual in its epilogue (and
 * RMSNorm runs as a kernel of its own after the output projection); more:
 * fp32 partials reduced with the residual (and RMSNorm) by one kernel.  Both
 * are 1 for fp32 dims or rows == 0.  Host arithmetic only. */
acache_status acache_layer_schedule(const acache_dims* dims, int32_t rows, int32_t* o_splits, int32_t* down_splits);

/* Workspace bytes needed by acache_layer_recompute, acache_score and
 * acache_linear for up to max_rows rows, `batch` requests and affix length
 * affix_len (0 when no scoring).  Returns 0 for invalid dims. */
size_t acache_workspace_size(const acache_dims* dims, int32_t max_rows, int32_t batch,
                             int32_t affix_len);

/* A static English description of a status code. */
const char* acache_status_string(acache_status status);

/* Library version, major * 10000 + minor * 100 + patch. */
int32_t acache_version(void);

#ifdef __cplusplus
}
#endif

#endif /* ACACHE_H */
