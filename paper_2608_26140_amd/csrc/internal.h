// Internal launch interface between the C ABI (api.cpp) and the gfx950
// kernels.  Every launcher enqueues on `stream` and returns the launch
// status; none allocates or synchronises.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/acache.h"

namespace acache {

constexpr int kMaxBatch = 64;

// Per-request row/key offsets and query-tile starts, passed by value.
struct Ragged {
  int batch;
  int cu_rows[kMaxBatch + 1];
  int cu_keys[kMaxBatch + 1];
  int tile_start[kMaxBatch + 1];  // cumulative query tiles of `tile_rows` rows
};

// ---- rows, maps, selection (k_rows.hip, k_topk.hip)
hipError_t launch_gather_rows(const void* src, int64_t src_ld, int64_t src_rows, const int32_t* idx,
                              const int32_t* remap, int64_t remap_len, int n, int row_bytes,
                              void* dst, int64_t dst_ld, hipStream_t s);
hipError_t launch_kv_scatter(const void* k_src, const void* v_src, int64_t src_ld_bytes, int n,
                             const int32_t* slots, void* k_pool, void* v_pool,
                             int64_t pool_ld_bytes, int64_t n_slots, int row_bytes, hipStream_t s);
// paging NULL: the layout's flat slot plan
hipError_t launch_build_maps(const acache_layout& lay, const acache_paging* paging, int batch,
                             const int32_t* anchors, int k, int32_t* row_pos, int32_t* row_src,
                             int32_t* write_slots, int32_t* read_slots, int32_t* q_rows, hipStream_t s);
hipError_t launch_topk(const float* scores, int batch, int L, int k, int32_t* out, hipStream_t s);
hipError_t launch_rmsnorm(acache_dtype dt, const void* x, const void* g, void* y, int rows, int d,
                          float eps, hipStream_t s);
// x[m] += sum_s part[s][m] (bf16 x, fp32 partials [splits][M][d]); if y,
// y[m] = RMSNorm(x[m]) * g.
hipError_t launch_reduce_residual(void* x, const float* part, int splits, int M, int d,
                                  const void* g, void* y, float eps, hipStream_t s);
// q[rows[i]] = rotary(sum_s part[s][i], pos[rows[i]]) for the n rows of bf16
// queries with head_dim 128 (fp32 partials [splits][n][H * 128]).
// bf16 RMSNorm of gathered rows: y[i] = norm(x[src_rows[i]]) (zero for an
// index outside [0, n_src)); needs rmsnorm_rows_ok (d % 8 == 0, d <= 8192,
// 16-byte aligned x, g and y).
bool rmsnorm_rows_ok(const void* x, const void* g, const void* y, int d);
hipError_t launch_rmsnorm_rows(const void* x, int64_t n_src, const int32_t* src_rows, const void* g, void* y,
                               int rows, int d, float eps, hipStream_t s);
// cos and sin of pos[m] * theta_d for every row m < M and rotary pair d < 64
// (head_dim 128): table[(m * 64 + d) * 2 + {0, 1}].
hipError_t launch_rope_table(const int32_t* pos, int M, float rope_base, float* table, hipStream_t s);
hipError_t launch_q_rotary_reduce(const float* part, int splits, int n, int H, const int32_t* rows,
                                  const int32_t* pos, float rope_base, void* q, int64_t q_n_rows, hipStream_t s);
// scores[b, j] (+)= sum over the request's H partial rows of part[b][r][j], in
// a fixed order; init: write instead of add
hipError_t launch_head_reduce(const float* part, int batch, int H, int L, float* scores, int init,
                              hipStream_t s);

// ---- bf16 MFMA GEMM (k_gemm.hip).  C = X W^T, X [M, K], W [N, K].
enum GemmEpi { EPI_STORE = 0, EPI_ACCUM = 1, EPI_PARTIAL = 2, EPI_QKV = 3, EPI_SWIGLU = 4 };
struct GemmParams {
  const void* X;
  const void* W;
  int M, N, K;      // N: weight rows (for SWIGLU: 2F)
  int splits;       // k splits (EPI_PARTIAL only)
  void* C;          // STORE / ACCUM / SWIGLU output, [M, ldc]
  int64_t ldc;
  float* P;         // PARTIAL output [splits][M][N]
  float* sk_ws;     // stream-K partials, gemm_bf16_sk_ws_bytes(); null: data-parallel only
  // QKV epilogue
  void* q_out;      // [M, hq_cols]
  void* k_pool;
  void* v_pool;
  int64_t pool_ld;
  int64_t n_slots;
  const int32_t* write_slots;
  const float* rope_cs;  // [M][64][2]: cos, sin of row m's rotary angle for pair d (launch_rope_table)
  int hq_cols, hkv_cols;
};
hipError_t launch_gemm_bf16(GemmEpi epi, const GemmParams& p, hipStream_t s);
int gemm_bf16_splits(int M, int N, int K);  // split-K choice for EPI_PARTIAL
size_t gemm_bf16_sk_ws_bytes();             // stream-K workspace (any shape)

hipError_t launch_argmax_commit(acache_dtype dt, const void* x, int64_t ld, int rows, int n, int32_t* out,
                               float* conf, const int32_t* commit_pos, int32_t* ids, int64_t ids_len, hipStream_t s);
hipError_t launch_threshold_commit(int batch, int block, const int32_t* pick, const float* conf, float tau,
                                  int32_t* committed, const int32_t* commit_pos, int32_t* ids, int64_t ids_len,
                                  int32_t* count, hipStream_t s);

hipError_t launch_rerotate(acache_dtype dt, const void* src, int64_t src_ld, const int32_t* src_slots, void* dst,
                           int64_t dst_ld, const int32_t* dst_slots, const int32_t* delta, int n, int64_t n_slots,
                           int heads, int dh, float rope_base, hipStream_t s);

hipError_t launch_kv_deviation(acache_dtype dt, const void* kp, const void* vp, int64_t pool_ld, int64_t n_slots,
                              const int32_t* fresh, int64_t fresh_ld, const int32_t* stale, int batch, int L,
                              int width, float* scores, hipStream_t s);

// ---- bf16 attention and scoring (k_attention.hip, k_score.hip)
// part / part_bytes: optional fp32 space for key splits (null: one split)
// lse_aff (nullable): also the natural-log log-sum-exp over each request's
// keys [aff_begin, aff_begin + aff_len), written only where aff_begin is 0
// (the running softmax's state once those keys are in) and aff_len is a
// multiple of 64 (under key splits the merge kernel combines the splits'
// shares); *aff_done (nullable) tells whether it was written.
hipError_t launch_attention_bf16(const Ragged& rg, int H, int Hkv, const void* q,
                                 const int32_t* read_slots, const void* k_pool, const void* v_pool,
                                 int64_t pool_ld, int64_t n_slots, void* out, float* lse,
                                 float* part, size_t part_bytes, hipStream_t s, float* lse_aff = nullptr,
                                 int aff_begin = 0, int aff_len = 0, bool* aff_done = nullptr);
// Decode-step attention: the queries of all requests against the shared
// affix slots (each request's anchors masked out), then each request's
// queries against its private slots, merged.  mask: [batch][ceil(L / 64)]
// scratch.  Returns hipErrorInvalidValue if part_bytes cannot hold two
// partial sets.
hipError_t launch_attention_decode_bf16(int batch, int rows_per_req, int H, int Hkv, const void* q,
                                        const int32_t* affix_slots, int L, const int32_t* anchors, int k,
                                        const int32_t* private_slots, int private_len, const void* k_pool,
                                        const void* v_pool, int64_t pool_ld, int64_t n_slots, void* out,
                                        uint64_t* mask, float* part, size_t part_bytes, hipStream_t s);
// Eq. 4-5 for one layer in one launch: part[b][r][j] for r < *rows_per_request
// (heads x query splits) such that the layer's score of affix key j of
// request b is the sum over r in order.  row_lse: [q_n_rows, H] natural-log
// normaliser (full-softmax reading) or null (affix-only, computed).
// hipErrorInvalidValue if part_bytes cannot hold batch * H * L floats.
hipError_t launch_score_fused_bf16(int batch, const int* cu_q, int H, int Hkv, const void* q, int64_t q_ld,
                                   int64_t q_n_rows, const int32_t* q_rows, const void* k_pool, int64_t pool_ld,
                                   int64_t n_slots, const int32_t* affix_slots, int L, const float* row_lse,
                                   float* part, size_t part_bytes, int* rows_per_request, hipStream_t s);

// ---- fp32 VALU path (k_f32.hip)
hipError_t launch_gemm_f32(const float* X, const float* W, float* C, int64_t ldc, int M, int N,
                           int K, int accumulate, hipStream_t s);
hipError_t launch_rope_scatter_f32(const float* qkv, int M, int H, int Hkv, int dh,
                                   const int32_t* pos, float rope_base, float* q_out,
                                   const int32_t* write_slots, float* k_pool, float* v_pool,
                                   int64_t pool_ld, int64_t n_slots, hipStream_t s);
hipError_t launch_swiglu_f32(const float* gu, int M, int F, float* h, hipStream_t s);
hipError_t launch_attention_f32(const Ragged& rg, int H, int Hkv, int dh, const float* q,
                                const int32_t* read_slots, const float* k_pool,
                                const float* v_pool, int64_t pool_ld, int64_t n_slots, float* out,
                                float* lse, hipStream_t s);
hipError_t launch_score_lse_f32(int batch, const int* cu_q, int H, int Hkv, int dh, const float* q,
                                int64_t q_ld, int64_t q_n_rows, const int32_t* q_rows,
                                const float* k_pool, int64_t pool_ld, int64_t n_slots,
                                const int32_t* affix_slots, int L, float* lse_out, hipStream_t s);
hipError_t launch_score_colsum_f32(int batch, const int* cu_q, int H, int Hkv, int dh,
                                   const float* q, int64_t q_ld, int64_t q_n_rows,
                                   const int32_t* q_rows, const float* k_pool, int64_t pool_ld,
                                   int64_t n_slots, const int32_t* affix_slots, int L,
                                   const float* lse, int lse_by_qrow, float* part, hipStream_t s);

}  // namespace acache
