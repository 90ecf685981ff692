// C ABI of the selective affix-KV recompute path: argument validation,
// workspace layout and the launch sequence of each entry point.  Nothing
// here allocates device memory or synchronises the stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <mutex>

#include "internal.h"

using namespace acache;

namespace {

constexpr size_t kAlign = 256;

inline size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }
inline bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }
inline size_t elem_size(acache_dtype dt) { return dt == ACACHE_BF16 ? 2 : 4; }

#define CHECK(cond, code) \
  do {                    \
    if (!(cond)) return (code); \
  } while (0)

#define LAUNCH(expr)                                   \
  do {                                                 \
    if ((expr) != hipSuccess) return ACACHE_ERR_DEVICE; \
  } while (0)

// Opt-in measurement hook (acache_time_kernel): events around one kernel id.
struct KernelTimer {
  int kernel = ACACHE_K_NONE;
  hipEvent_t* starts = nullptr;
  hipEvent_t* stops = nullptr;
  int capacity = 0;
  int32_t* count = nullptr;
};
KernelTimer g_timer;

inline bool timed(int id) {
  return g_timer.kernel == id && g_timer.count && *g_timer.count < g_timer.capacity;
}

// LAUNCH with the kernel's start/stop events recorded when it is armed.
#define LAUNCH_T(id, strm, expr)                                                            \
  do {                                                                                      \
    const bool t_ = timed(id);                                                              \
    if (t_ && hipEventRecord(g_timer.starts[*g_timer.count], strm) != hipSuccess)           \
      return ACACHE_ERR_DEVICE;                                                             \
    if ((expr) != hipSuccess) return ACACHE_ERR_DEVICE;                                     \
    if (t_) {                                                                               \
      if (hipEventRecord(g_timer.stops[*g_timer.count], strm) != hipSuccess) return ACACHE_ERR_DEVICE; \
      ++*g_timer.count;                                                                     \
    }                                                                                       \
  } while (0)

acache_status check_dims(const acache_dims* d) {
  CHECK(d, ACACHE_ERR_NULL);
  CHECK(d->dtype == ACACHE_BF16 || d->dtype == ACACHE_F32, ACACHE_ERR_UNSUPPORTED);
  CHECK(d->d_model > 0 && d->n_heads > 0 && d->n_kv_heads > 0 && d->head_dim > 0 && d->d_ff > 0,
        ACACHE_ERR_SHAPE);
  CHECK(d->n_heads % d->n_kv_heads == 0, ACACHE_ERR_SHAPE);
  CHECK(d->rms_eps >= 0.f && d->rope_base > 0.f, ACACHE_ERR_SHAPE);
  if (d->dtype == ACACHE_BF16) {
    CHECK(d->head_dim == 128, ACACHE_ERR_UNSUPPORTED);
  } else {
    CHECK(d->head_dim % 2 == 0 && d->head_dim <= 128, ACACHE_ERR_UNSUPPORTED);
  }
  return ACACHE_OK;
}

// Shapes the bf16 GEMM tiles and the fused epilogues need.
acache_status check_layer_dims(const acache_dims* d) {
  acache_status st = check_dims(d);
  if (st != ACACHE_OK) return st;
  if (d->dtype == ACACHE_BF16) {
    CHECK(d->d_model % 256 == 0 && d->d_model <= 8192, ACACHE_ERR_UNSUPPORTED);
    CHECK((d->n_heads * d->head_dim) % 256 == 0, ACACHE_ERR_UNSUPPORTED);
    CHECK((d->n_kv_heads * d->head_dim) % 128 == 0, ACACHE_ERR_UNSUPPORTED);
    CHECK(((d->n_heads + 2 * d->n_kv_heads) * d->head_dim) % 256 == 0, ACACHE_ERR_UNSUPPORTED);
    CHECK(d->d_ff % 128 == 0, ACACHE_ERR_UNSUPPORTED);
  }
  return ACACHE_OK;
}

// Validates host cu arrays and fills the kernel-side copy.
acache_status make_ragged(const acache_ragged* rg, Ragged& out) {
  CHECK(rg && rg->cu_rows && rg->cu_keys, ACACHE_ERR_NULL);
  CHECK(rg->batch >= 1 && rg->batch <= kMaxBatch, ACACHE_ERR_SHAPE);
  CHECK(rg->cu_rows[0] == 0 && rg->cu_keys[0] == 0, ACACHE_ERR_SHAPE);
  std::memset(&out, 0, sizeof(out));
  out.batch = rg->batch;
  for (int b = 0; b <= rg->batch; ++b) {
    out.cu_rows[b] = rg->cu_rows[b];
    out.cu_keys[b] = rg->cu_keys[b];
    if (b > 0) {
      const int nr = rg->cu_rows[b] - rg->cu_rows[b - 1];
      const int nk = rg->cu_keys[b] - rg->cu_keys[b - 1];
      CHECK(nr >= 0 && nk >= 0, ACACHE_ERR_SHAPE);
      CHECK(nr == 0 || nk > 0, ACACHE_ERR_SHAPE);  // rows need keys
    }
  }
  return ACACHE_OK;
}

acache_status check_cu(const int32_t* cu, int batch) {
  CHECK(cu, ACACHE_ERR_NULL);
  CHECK(cu[0] == 0, ACACHE_ERR_SHAPE);
  for (int b = 1; b <= batch; ++b) CHECK(cu[b] >= cu[b - 1], ACACHE_ERR_SHAPE);
  return ACACHE_OK;
}

// Workspace plan for `rows` rows (layer_recompute / score / linear).
struct WsPlan {
  size_t y, q, o, h, part, qkv, gu, rope, lse, lse_aff, colsum, colsum_bytes, total;
  size_t part_bytes;  // size of the part region (split-K / stream-K / attention key-split partials)
};

WsPlan plan_ws(const acache_dims* d, int rows, int batch, int L) {
  WsPlan w = {};
  const size_t es = elem_size(d->dtype);
  const size_t M = (size_t)rows;
  const size_t hq = (size_t)d->n_heads * d->head_dim;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += align_up(bytes);
    return at;
  };
  w.y = take(M * d->d_model * es);
  w.q = take(M * hq * es);
  w.o = take(M * hq * es);
  w.h = take(M * d->d_ff * es);
  if (d->dtype == ACACHE_BF16) {
    // largest splits x rows over every row count up to `rows`, so one
    // workspace serves any smaller call (splits change only at row-tile
    // boundaries, every one of which is a multiple of 128 rows)
    size_t part_elems = 0;
    for (int t = 1; (t - 1) * 128 < rows; ++t) {
      const int m = std::min(rows, t * 128);
      const int sp = std::max(gemm_bf16_splits(m, d->d_model, (int)hq), gemm_bf16_splits(m, d->d_model, d->d_ff));
      part_elems = std::max(part_elems, (size_t)sp * (size_t)m * d->d_model);
      // the query-only projection of the probe's last layer
      part_elems = std::max(part_elems, (size_t)gemm_bf16_splits(m, (int)hq, d->d_model) * (size_t)m * hq);
    }
    // split-K partials of the O / down projections and the stream-K pieces
    // of the QKV / gate-up projections are never live at the same time
    w.part_bytes = std::max(part_elems * sizeof(float), gemm_bf16_sk_ws_bytes());
    w.part = take(w.part_bytes);
    w.qkv = w.gu = 0;
    // the rotary table of the QKV projection: (cos, sin) of 64 pairs per row
    w.rope = take(M * 64 * 2 * sizeof(float));
  } else {
    w.qkv = take(M * (size_t)(d->n_heads + 2 * d->n_kv_heads) * d->head_dim * es);
    w.gu = take(M * 2 * (size_t)d->d_ff * es);
    w.part = 0;
    w.rope = 0;
  }
  w.lse = take(M * d->n_heads * sizeof(float));
  w.lse_aff = take(M * d->n_heads * sizeof(float));
  // column sums per head and per query split (up to 8 splits at this size;
  // the scoring kernel takes as many as fit)
  w.colsum_bytes = (size_t)(batch > 0 ? batch : 1) * d->n_heads * (size_t)(L > 0 ? L : 1) * sizeof(float) * 8;
  w.colsum = take(w.colsum_bytes);
  w.total = off;
  return w;
}

template <typename T>
T* at(void* ws, size_t off) {
  return reinterpret_cast<T*>(static_cast<char*>(ws) + off);
}

// Eq. 4-5 for one layer (shared by acache_score and the probe mode of
// acache_layer_recompute).  lse_full: [q_n_rows, H] natural log, or NULL.
// colsum: colsum_bytes of scratch for the per-head (and per-split) column
// sums; lse_aff: [q_n_rows, H] scratch of the fp32 path.  aff_given
// (nullable, bf16): the rows' log-sum-exp over the affix keys already taken
// (by the layer's attention), used instead of the score's own pass.
acache_status run_score(const acache_dims* d, int batch, const int32_t* cu_q, const void* q,
                        int64_t q_ld, int64_t q_n_rows, const int32_t* q_rows, const void* k_pool,
                        int64_t pool_ld, int64_t n_slots, const int32_t* affix_slots, int L,
                        acache_norm norm, const float* lse_full, float* scores, float* lse_aff,
                        float* colsum, size_t colsum_bytes, int init, hipStream_t s,
                        const float* aff_given = nullptr) {
  const int H = d->n_heads, Hkv = d->n_kv_heads, dh = d->head_dim;
  if (d->dtype == ACACHE_BF16) {
    int rows = H;
    LAUNCH_T(ACACHE_K_SCORE_COLSUM, s,
             launch_score_fused_bf16(batch, cu_q, H, Hkv, q, q_ld, q_n_rows, q_rows, k_pool, pool_ld, n_slots,
                                     affix_slots, L, norm == ACACHE_NORM_FULL ? lse_full : aff_given, colsum,
                                     colsum_bytes, &rows, s));
    LAUNCH_T(ACACHE_K_SCORE_REDUCE, s, launch_head_reduce(colsum, batch, rows, L, scores, init, s));
    return ACACHE_OK;
  }
  const float* lse = lse_full;
  int by_qrow = 0;
  if (norm == ACACHE_NORM_AFFIX) {
    LAUNCH_T(ACACHE_K_SCORE_LSE, s, launch_score_lse_f32(batch, cu_q, H, Hkv, dh, (const float*)q, q_ld, q_n_rows, q_rows,
                                (const float*)k_pool, pool_ld, n_slots, affix_slots, L, lse_aff, s));
    lse = lse_aff;
    by_qrow = 1;
  }
  LAUNCH_T(ACACHE_K_SCORE_COLSUM, s, launch_score_colsum_f32(batch, cu_q, H, Hkv, dh, (const float*)q, q_ld, q_n_rows, q_rows,
                                 (const float*)k_pool, pool_ld, n_slots, affix_slots, L, lse, by_qrow,
                                 colsum, s));
  LAUNCH_T(ACACHE_K_SCORE_REDUCE, s, launch_head_reduce(colsum, batch, H, L, scores, init, s));
  return ACACHE_OK;
}

// Device memory of acache_score_noalloc: the library's own fixed scratch
// (one copy per GPU, held until the process ends).  Host code never names
// the array directly: its device address comes from hipGetSymbolAddress,
// once per device, on the first call on that device.
constexpr size_t kNoallocScratchBytes = size_t(64) << 20;
__device__ __align__(256) char scratch[kNoallocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's scratch address, resolved on its first use.
acache_status scratch_address(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return ACACHE_ERR_DEVICE;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return ACACHE_ERR_DEVICE;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return ACACHE_OK;
}

}  // namespace

extern "C" {

int32_t acache_version(void) { return 100; }

const char* acache_status_string(acache_status st) {
  switch (st) {
    case ACACHE_OK: return "ok";
    case ACACHE_ERR_NULL: return "a required pointer is NULL";
    case ACACHE_ERR_SHAPE: return "sizes are negative, inconsistent or out of range";
    case ACACHE_ERR_ALIGN: return "a pointer or leading dimension is not 16-byte aligned";
    case ACACHE_ERR_UNSUPPORTED: return "shape or type outside what the kernels implement";
    case ACACHE_ERR_WORKSPACE: return "workspace missing or too small";
    case ACACHE_ERR_DEVICE: return "a HIP launch or call failed";
    case ACACHE_ERR_SPACE: return "not enough free blocks in the pool";
  }
  return "unknown status";
}

acache_status acache_time_kernel(int32_t kernel, hipEvent_t* starts, hipEvent_t* stops,
                                 int32_t capacity, int32_t* count) {
  if (kernel == ACACHE_K_NONE) {
    g_timer = KernelTimer();
    return ACACHE_OK;
  }
  CHECK(kernel >= 0 && kernel < ACACHE_K_COUNT && capacity >= 0, ACACHE_ERR_SHAPE);
  CHECK(count && (capacity == 0 || (starts && stops)), ACACHE_ERR_NULL);
  g_timer.kernel = kernel;
  g_timer.starts = starts;
  g_timer.stops = stops;
  g_timer.capacity = capacity;
  g_timer.count = count;
  return ACACHE_OK;
}

size_t acache_workspace_size(const acache_dims* dims, int32_t max_rows, int32_t batch,
                             int32_t affix_len) {
  if (check_dims(dims) != ACACHE_OK || max_rows < 0 || batch < 0 || affix_len < 0) return 0;
  return plan_ws(dims, max_rows, batch, affix_len).total;
}

int32_t acache_anchor_count(double ratio, int32_t affix_len) {
  if (!(ratio >= 0.0 && ratio <= 1.0) || affix_len < 0) return -1;
  // ratio * L is exact in double for L < 2^31 up to the product's rounding;
  // the half-up rule is floor(x + 1/2)
  const double k = std::floor(ratio * (double)affix_len + 0.5);
  return (int32_t)std::min<double>(std::max(k, 0.0), (double)affix_len);
}

acache_status acache_topk(const float* scores, int32_t batch, int32_t L, int32_t k,
                          int32_t* idx_out, hipStream_t stream) {
  CHECK(batch >= 0 && L >= 0 && k >= 0 && k <= L, ACACHE_ERR_SHAPE);
  CHECK(L <= 16384, ACACHE_ERR_UNSUPPORTED);
  if (batch == 0 || k == 0) return ACACHE_OK;
  CHECK(scores && idx_out, ACACHE_ERR_NULL);
  LAUNCH_T(ACACHE_K_TOPK, stream, launch_topk(scores, batch, L, k, idx_out, stream));
  return ACACHE_OK;
}

acache_status acache_gather_rows(const void* src, int64_t src_ld_bytes, int64_t src_rows,
                                 const int32_t* idx, const int32_t* remap, int64_t remap_len,
                                 int32_t n, int32_t row_bytes, void* dst, int64_t dst_ld_bytes,
                                 hipStream_t stream) {
  CHECK(n >= 0 && row_bytes >= 0 && src_rows >= 0, ACACHE_ERR_SHAPE);
  if (n == 0 || row_bytes == 0) return ACACHE_OK;
  CHECK(src && idx && dst, ACACHE_ERR_NULL);
  CHECK(row_bytes % 16 == 0 && src_ld_bytes >= row_bytes && dst_ld_bytes >= row_bytes, ACACHE_ERR_SHAPE);
  CHECK(!remap || remap_len >= 0, ACACHE_ERR_SHAPE);
  CHECK(aligned16(src) && aligned16(dst) && src_ld_bytes % 16 == 0 && dst_ld_bytes % 16 == 0,
        ACACHE_ERR_ALIGN);
  LAUNCH_T(ACACHE_K_GATHER, stream, launch_gather_rows(src, src_ld_bytes, src_rows, idx, remap, remap_len, n, row_bytes, dst,
                            dst_ld_bytes, stream));
  return ACACHE_OK;
}

acache_status acache_kv_scatter(const void* k_src, const void* v_src, int64_t src_ld, int32_t n,
                                const int32_t* dst_slots, void* k_pool, void* v_pool,
                                int64_t pool_ld, int64_t n_slots, int32_t row_elems,
                                acache_dtype dtype, hipStream_t stream) {
  CHECK(dtype == ACACHE_BF16 || dtype == ACACHE_F32, ACACHE_ERR_UNSUPPORTED);
  CHECK(n >= 0 && row_elems >= 0 && n_slots >= 0, ACACHE_ERR_SHAPE);
  if (n == 0 || row_elems == 0) return ACACHE_OK;
  CHECK(k_src && v_src && dst_slots && k_pool && v_pool, ACACHE_ERR_NULL);
  const int64_t es = (int64_t)elem_size(dtype);
  CHECK(src_ld >= row_elems && pool_ld >= row_elems, ACACHE_ERR_SHAPE);
  CHECK((row_elems * es) % 16 == 0, ACACHE_ERR_SHAPE);
  CHECK(aligned16(k_src) && aligned16(v_src) && aligned16(k_pool) && aligned16(v_pool) &&
            (src_ld * es) % 16 == 0 && (pool_ld * es) % 16 == 0,
        ACACHE_ERR_ALIGN);
  LAUNCH_T(ACACHE_K_SCATTER, stream, launch_kv_scatter(k_src, v_src, src_ld * es, n, dst_slots, k_pool, v_pool, pool_ld * es,
                           n_slots, (int)(row_elems * es), stream));
  return ACACHE_OK;
}

acache_status acache_rerotate_k(const acache_dims* dims, const void* k_src, const int32_t* src_slots, void* k_dst,
                                const int32_t* dst_slots, const int32_t* delta, int32_t n, int64_t pool_ld,
                                int64_t n_slots, hipStream_t stream) {
  acache_status st = check_dims(dims);
  if (st != ACACHE_OK) return st;
  CHECK(n >= 0 && n_slots >= 0, ACACHE_ERR_SHAPE);
  if (n == 0) return ACACHE_OK;
  CHECK(k_src && src_slots && k_dst && dst_slots && delta, ACACHE_ERR_NULL);
  CHECK(pool_ld >= (int64_t)dims->n_kv_heads * dims->head_dim, ACACHE_ERR_SHAPE);
  LAUNCH(launch_rerotate(dims->dtype, k_src, pool_ld, src_slots, k_dst, pool_ld, dst_slots, delta, n, n_slots,
                         dims->n_kv_heads, dims->head_dim, dims->rope_base, stream));
  return ACACHE_OK;
}

acache_status acache_kv_deviation(const acache_dims* dims, int32_t batch, int32_t affix_len, const void* k_pool,
                                  const void* v_pool, int64_t pool_ld, int64_t n_slots, const int32_t* fresh_slots,
                                  int64_t fresh_ld, const int32_t* stale_slots, float* scores, hipStream_t stream) {
  acache_status st = check_dims(dims);
  if (st != ACACHE_OK) return st;
  CHECK(batch >= 0 && batch <= 65535 && affix_len >= 0 && fresh_ld >= affix_len, ACACHE_ERR_SHAPE);
  if (batch == 0 || affix_len == 0) return ACACHE_OK;
  CHECK(k_pool && v_pool && fresh_slots && stale_slots && scores, ACACHE_ERR_NULL);
  const int64_t width = (int64_t)dims->n_kv_heads * dims->head_dim;
  const int64_t es = (int64_t)elem_size(dims->dtype);
  CHECK(pool_ld >= width && (width * es) % 16 == 0, ACACHE_ERR_SHAPE);
  CHECK(aligned16(k_pool) && aligned16(v_pool) && (pool_ld * es) % 16 == 0, ACACHE_ERR_ALIGN);
  LAUNCH(launch_kv_deviation(dims->dtype, k_pool, v_pool, pool_ld, n_slots, fresh_slots, fresh_ld, stale_slots,
                             batch, affix_len, (int)width, scores, stream));
  return ACACHE_OK;
}

acache_status acache_argmax_commit(acache_dtype dtype, const void* x, int64_t ld, int32_t rows, int32_t n,
                                   int32_t* out, float* conf, const int32_t* commit_pos, int32_t* ids,
                                   int64_t ids_len, hipStream_t stream) {
  CHECK(dtype == ACACHE_BF16 || dtype == ACACHE_F32, ACACHE_ERR_UNSUPPORTED);
  CHECK(rows >= 0 && n >= 0 && ld >= n && ids_len >= 0, ACACHE_ERR_SHAPE);
  if (rows == 0) return ACACHE_OK;
  CHECK(n > 0, ACACHE_ERR_SHAPE);
  CHECK(x && out && (!commit_pos || ids), ACACHE_ERR_NULL);
  LAUNCH_T(ACACHE_K_ARGMAX, stream, launch_argmax_commit(dtype, x, ld, rows, n, out, conf, commit_pos, ids, ids_len, stream));
  return ACACHE_OK;
}

acache_status acache_threshold_commit(int32_t batch, int32_t block, const int32_t* pick, const float* conf, float tau,
                                      int32_t* committed, const int32_t* commit_pos, int32_t* ids, int64_t ids_len,
                                      int32_t* count, hipStream_t stream) {
  CHECK(batch >= 0 && block >= 0 && ids_len >= 0, ACACHE_ERR_SHAPE);
  if (batch == 0) return ACACHE_OK;
  CHECK(pick && conf && committed && commit_pos && ids && count, ACACHE_ERR_NULL);
  LAUNCH(launch_threshold_commit(batch, block, pick, conf, tau, committed, commit_pos, ids, ids_len, count, stream));
  return ACACHE_OK;
}

static acache_status check_layout(const acache_layout* lay, int32_t batch, int32_t k) {
  CHECK(lay, ACACHE_ERR_NULL);
  const int S = lay->seq_len, ab = lay->affix_begin, L = lay->affix_len;
  CHECK(batch >= 0 && S >= 0 && L >= 0 && ab >= 0 && ab + L <= S, ACACHE_ERR_SHAPE);
  CHECK(k >= 0 && k <= L, ACACHE_ERR_SHAPE);
  CHECK(lay->mask_len >= 0 && lay->mask_begin >= 0 && lay->mask_begin + lay->mask_len <= S,
        ACACHE_ERR_SHAPE);
  CHECK(lay->mask_len == 0 || lay->mask_begin + lay->mask_len <= ab || lay->mask_begin >= ab + L,
        ACACHE_ERR_SHAPE);  // the masked span is not part of the affix
  CHECK((int64_t)batch * S < (int64_t)1 << 31, ACACHE_ERR_SHAPE);
  CHECK(lay->key_order == 0 || lay->key_order == 1, ACACHE_ERR_UNSUPPORTED);
  return ACACHE_OK;
}

acache_status acache_build_maps_paged(const acache_layout* lay, const acache_paging* paging, int32_t batch,
                                      const int32_t* anchors, int32_t k, int32_t* row_pos, int32_t* row_src,
                                      int32_t* write_slots, int32_t* read_slots, int32_t* q_rows,
                                      hipStream_t stream) {
  acache_status st = check_layout(lay, batch, k);
  if (st != ACACHE_OK) return st;
  CHECK(paging, ACACHE_ERR_NULL);
  const int R = k + lay->seq_len - lay->affix_len;
  CHECK(paging->block_size >= 1 && paging->blocks_per_request >= 0, ACACHE_ERR_SHAPE);
  CHECK((int64_t)paging->blocks_per_request * paging->block_size >= R, ACACHE_ERR_SHAPE);
  if (batch == 0 || lay->seq_len == 0) return ACACHE_OK;
  CHECK(row_pos && row_src && write_slots && read_slots, ACACHE_ERR_NULL);
  CHECK(k == 0 || anchors, ACACHE_ERR_NULL);
  CHECK(lay->affix_len == k || paging->shared_blocks, ACACHE_ERR_NULL);  // some affix position reads shared
  CHECK(R == 0 || paging->private_blocks, ACACHE_ERR_NULL);
  LAUNCH_T(ACACHE_K_MAPS, stream, launch_build_maps(*lay, paging, batch, anchors, k, row_pos, row_src, write_slots,
                                                    read_slots, q_rows, stream));
  return ACACHE_OK;
}

acache_status acache_build_maps(const acache_layout* lay, int32_t batch, const int32_t* anchors,
                                int32_t k, int32_t* row_pos, int32_t* row_src,
                                int32_t* write_slots, int32_t* read_slots, int32_t* q_rows,
                                hipStream_t stream) {
  acache_status st = check_layout(lay, batch, k);
  if (st != ACACHE_OK) return st;
  const int S = lay->seq_len, L = lay->affix_len;
  const int R = k + S - L;
  CHECK(lay->private_stride >= R && lay->private_base >= 0 && lay->shared_base >= 0, ACACHE_ERR_SHAPE);
  CHECK((int64_t)lay->private_base + (int64_t)batch * lay->private_stride < (int64_t)1 << 31,
        ACACHE_ERR_SHAPE);
  if (batch == 0 || S == 0) return ACACHE_OK;
  CHECK(row_pos && row_src && write_slots && read_slots, ACACHE_ERR_NULL);
  CHECK(k == 0 || anchors, ACACHE_ERR_NULL);
  LAUNCH_T(ACACHE_K_MAPS, stream, launch_build_maps(*lay, nullptr, batch, anchors, k, row_pos, row_src, write_slots,
                                                    read_slots, q_rows, stream));
  return ACACHE_OK;
}

acache_status acache_rmsnorm(const acache_dims* dims, const void* x, const void* g, void* y,
                             int32_t rows, hipStream_t stream) {
  acache_status st = check_dims(dims);
  if (st != ACACHE_OK) return st;
  CHECK(rows >= 0, ACACHE_ERR_SHAPE);
  if (rows == 0) return ACACHE_OK;
  CHECK(x && g && y, ACACHE_ERR_NULL);
  LAUNCH(launch_rmsnorm(dims->dtype, x, g, y, rows, dims->d_model, dims->rms_eps, stream));
  return ACACHE_OK;
}

acache_status acache_linear(const acache_dims* dims, const void* a, const void* w, void* c,
                            int32_t M, int32_t N, int32_t K, int32_t accumulate, void* ws,
                            size_t ws_bytes, hipStream_t stream) {
  CHECK(dims, ACACHE_ERR_NULL);
  CHECK(dims->dtype == ACACHE_BF16 || dims->dtype == ACACHE_F32, ACACHE_ERR_UNSUPPORTED);
  CHECK(M >= 0 && N >= 0 && K >= 0, ACACHE_ERR_SHAPE);
  if (M == 0 || N == 0) return ACACHE_OK;
  CHECK(a && w && c, ACACHE_ERR_NULL);
  // operands are addressed with 32-bit element offsets
  CHECK((int64_t)M * K < ((int64_t)1 << 31) && (int64_t)N * K < ((int64_t)1 << 31), ACACHE_ERR_UNSUPPORTED);
  if (dims->dtype == ACACHE_BF16) {
    CHECK(K > 0 && K % 64 == 0 && N % 256 == 0, ACACHE_ERR_UNSUPPORTED);
    CHECK(aligned16(a) && aligned16(w) && aligned16(c), ACACHE_ERR_ALIGN);
    GemmParams p = {};
    p.X = a;
    p.W = w;
    p.M = M;
    p.N = N;
    p.K = K;
    p.splits = 1;
    p.C = c;
    p.ldc = N;
    // a workspace large enough for the stream-K partials enables stream-K
    if (ws && aligned16(ws) && ws_bytes >= gemm_bf16_sk_ws_bytes()) p.sk_ws = (float*)ws;
    LAUNCH(launch_gemm_bf16(accumulate ? EPI_ACCUM : EPI_STORE, p, stream));
  } else {
    LAUNCH(launch_gemm_f32((const float*)a, (const float*)w, (float*)c, N, M, N, K, accumulate, stream));
  }
  return ACACHE_OK;
}

acache_status acache_attention(const acache_dims* dims, const acache_ragged* rg, const void* q,
                               const int32_t* read_slots, const void* k_pool, const void* v_pool,
                               int64_t pool_ld, int64_t n_slots, void* out, float* lse,
                               hipStream_t stream) {
  acache_status st = check_dims(dims);
  if (st != ACACHE_OK) return st;
  Ragged r;
  st = make_ragged(rg, r);
  if (st != ACACHE_OK) return st;
  const int rows = r.cu_rows[r.batch];
  if (rows == 0) return ACACHE_OK;
  CHECK(q && read_slots && k_pool && v_pool && out, ACACHE_ERR_NULL);
  CHECK(pool_ld >= (int64_t)dims->n_kv_heads * dims->head_dim && n_slots >= 0, ACACHE_ERR_SHAPE);
  CHECK(n_slots * pool_ld < ((int64_t)1 << 31), ACACHE_ERR_UNSUPPORTED);  // 32-bit element offsets
  const int64_t es = (int64_t)elem_size(dims->dtype);
  CHECK(aligned16(q) && aligned16(k_pool) && aligned16(v_pool) && aligned16(out) && (pool_ld * es) % 16 == 0,
        ACACHE_ERR_ALIGN);
  if (dims->dtype == ACACHE_BF16)
    LAUNCH_T(ACACHE_K_ATTENTION, stream, launch_attention_bf16(r, dims->n_heads, dims->n_kv_heads, q, read_slots, k_pool, v_pool,
                                 pool_ld, n_slots, out, lse, nullptr, 0, stream));
  else
    LAUNCH_T(ACACHE_K_ATTENTION, stream, launch_attention_f32(r, dims->n_heads, dims->n_kv_heads, dims->head_dim, (const float*)q,
                                read_slots, (const float*)k_pool, (const float*)v_pool, pool_ld, n_slots,
                                (float*)out, lse, stream));
  return ACACHE_OK;
}

// Host checks of acache_score and acache_score_noalloc.  Sets *noop when the
// call has nothing to do.
static acache_status check_score(const acache_dims* dims, int32_t batch, const void* q, int64_t q_ld,
                                 int64_t q_n_rows, const int32_t* q_rows, const int32_t* cu_q, const void* k_pool,
                                 int64_t pool_ld, int64_t n_slots, const int32_t* affix_slots, int32_t affix_len,
                                 const float* row_lse, acache_norm norm, const float* scores, bool* noop) {
  *noop = true;
  acache_status st = check_dims(dims);
  if (st != ACACHE_OK) return st;
  CHECK(batch >= 0 && batch <= kMaxBatch && affix_len >= 0 && affix_len <= 65536, ACACHE_ERR_SHAPE);
  CHECK(norm == ACACHE_NORM_AFFIX || norm == ACACHE_NORM_FULL, ACACHE_ERR_UNSUPPORTED);
  if (batch == 0 || affix_len == 0) return ACACHE_OK;
  st = check_cu(cu_q, batch);
  if (st != ACACHE_OK) return st;
  if (cu_q[batch] == 0) return ACACHE_OK;
  CHECK(q && q_rows && k_pool && affix_slots && scores, ACACHE_ERR_NULL);
  CHECK(norm == ACACHE_NORM_FULL ? row_lse != nullptr : row_lse == nullptr, ACACHE_ERR_NULL);
  CHECK(q_ld >= (int64_t)dims->n_heads * dims->head_dim && q_n_rows >= 0, ACACHE_ERR_SHAPE);
  CHECK(pool_ld >= (int64_t)dims->n_kv_heads * dims->head_dim && n_slots >= 0, ACACHE_ERR_SHAPE);
  CHECK(n_slots * pool_ld < ((int64_t)1 << 31), ACACHE_ERR_UNSUPPORTED);  // 32-bit element offsets
  const int64_t es = (int64_t)elem_size(dims->dtype);
  CHECK(aligned16(q) && aligned16(k_pool) && (q_ld * es) % 16 == 0 && (pool_ld * es) % 16 == 0,
        ACACHE_ERR_ALIGN);
  *noop = false;
  return ACACHE_OK;
}

acache_status acache_score(const acache_dims* dims, int32_t batch, const void* q, int64_t q_ld,
                           int64_t q_n_rows, const int32_t* q_rows, const int32_t* cu_q,
                           const void* k_pool, int64_t pool_ld, int64_t n_slots,
                           const int32_t* affix_slots, int32_t affix_len, const float* row_lse,
                           acache_norm norm, float* scores, void* ws, size_t ws_bytes,
                           hipStream_t stream) {
  bool noop = true;
  acache_status st = check_score(dims, batch, q, q_ld, q_n_rows, q_rows, cu_q, k_pool, pool_ld, n_slots,
                                 affix_slots, affix_len, row_lse, norm, scores, &noop);
  if (st != ACACHE_OK || noop) return st;
  // workspace: the lse and column-sum regions of a plan sized for n_q rows
  const WsPlan w = plan_ws(dims, cu_q[batch], batch, affix_len);
  CHECK(ws && ws_bytes >= w.total, ACACHE_ERR_WORKSPACE);
  return run_score(dims, batch, cu_q, q, q_ld, q_n_rows, q_rows, k_pool, pool_ld, n_slots, affix_slots,
                   affix_len, norm, row_lse, scores, at<float>(ws, w.lse_aff), at<float>(ws, w.colsum),
                   w.colsum_bytes, 0, stream);
}

acache_status acache_score_noalloc(const acache_dims* dims, int32_t batch, const void* q, int64_t q_ld,
                                   int64_t q_n_rows, const int32_t* q_rows, const int32_t* cu_q,
                                   const void* k_pool, int64_t pool_ld, int64_t n_slots,
                                   const int32_t* affix_slots, int32_t affix_len, const float* row_lse,
                                   acache_norm norm, float* scores, hipStream_t stream) {
  bool noop = true;
  acache_status st = check_score(dims, batch, q, q_ld, q_n_rows, q_rows, cu_q, k_pool, pool_ld, n_slots,
                                 affix_slots, affix_len, row_lse, norm, scores, &noop);
  if (st != ACACHE_OK || noop) return st;
  // the lse and column-sum regions, laid out as in a workspace, must fit the
  // fixed scratch; both are written in full before they are read, so the
  // previous call's contents need no clearing
  const size_t lse_bytes = align_up((size_t)cu_q[batch] * dims->n_heads * sizeof(float));
  const size_t colsum_bytes = align_up((size_t)batch * dims->n_heads * (size_t)affix_len * sizeof(float));
  CHECK(lse_bytes + colsum_bytes <= kNoallocScratchBytes, ACACHE_ERR_WORKSPACE);
  void* base = nullptr;
  st = scratch_address(&base);
  if (st != ACACHE_OK) return st;
  return run_score(dims, batch, cu_q, q, q_ld, q_n_rows, q_rows, k_pool, pool_ld, n_slots, affix_slots,
                   affix_len, norm, row_lse, scores, at<float>(base, 0), at<float>(base, lse_bytes),
                   kNoallocScratchBytes - lse_bytes, 0, stream);
}

size_t acache_score_noalloc_max_bytes(void) { return kNoallocScratchBytes; }

acache_status acache_layer_schedule(const acache_dims* dims, int32_t rows, int32_t* o_splits, int32_t* down_splits) {
  acache_status st = check_layer_dims(dims);
  if (st != ACACHE_OK) return st;
  CHECK(rows >= 0, ACACHE_ERR_SHAPE);
  CHECK(o_splits && down_splits, ACACHE_ERR_NULL);
  const int d = dims->d_model, hq = dims->n_heads * dims->head_dim;
  if (dims->dtype != ACACHE_BF16 || rows == 0) {
    *o_splits = *down_splits = 1;
    return ACACHE_OK;
  }
  *o_splits = gemm_bf16_splits(rows, d, hq);
  *down_splits = gemm_bf16_splits(rows, d, dims->d_ff);
  return ACACHE_OK;
}

// bf16 block pieces shared by acache_layer_recompute and acache_layer_decode.
// QKV projection of the normalised rows y with rotary embedding; Q to q, the
// fresh K/V to their pool slots.
static acache_status run_qkv_bf16(const acache_dims* dims, const acache_layer_weights* w, int M, const void* y,
                                  void* q, const int32_t* pos, const int32_t* write_slots, void* k_pool,
                                  void* v_pool, int64_t pool_ld, int64_t n_slots, float* part, float* rope,
                                  hipStream_t stream) {
  const int d = dims->d_model, H = dims->n_heads, Hkv = dims->n_kv_heads, dh = dims->head_dim;
  LAUNCH(launch_rope_table(pos, M, dims->rope_base, rope, stream));
  GemmParams g = {};
  g.X = y;
  g.W = w->w_qkv;
  g.M = M;
  g.N = (H + 2 * Hkv) * dh;
  g.K = d;
  g.splits = 1;
  g.q_out = q;
  g.k_pool = k_pool;
  g.v_pool = v_pool;
  g.pool_ld = pool_ld;
  g.n_slots = n_slots;
  g.write_slots = write_slots;
  g.rope_cs = rope;
  g.hq_cols = H * dh;
  g.hkv_cols = Hkv * dh;
  g.sk_ws = part;
  LAUNCH_T(ACACHE_K_GEMM_QKV, stream, launch_gemm_bf16(EPI_QKV, g, stream));
  return ACACHE_OK;
}

// O projection + residual + RMSNorm, SwiGLU MLP + residual, from the
// attention output o; x is updated in place, y and hb are scratch.
static acache_status run_out_mlp_bf16(const acache_dims* dims, const acache_layer_weights* w, int M, void* x,
                                      void* y, const void* o, void* hb, float* part, hipStream_t stream) {
  const int d = dims->d_model, hq = dims->n_heads * dims->head_dim, F = dims->d_ff;
  GemmParams g = {};
  g.X = o;
  g.W = w->w_o;
  g.M = M;
  g.N = d;
  g.K = hq;
  g.splits = gemm_bf16_splits(M, d, hq);
  if (g.splits == 1) {
    // one K split: the projection adds itself to the residual in its
    // epilogue (x + acc rounded once, as the reduction would), then RMSNorm
    g.splits = 1;
    g.C = x;
    g.ldc = d;
    g.sk_ws = part;
    LAUNCH_T(ACACHE_K_GEMM_O, stream, launch_gemm_bf16(EPI_ACCUM, g, stream));
    LAUNCH_T(ACACHE_K_RMSNORM, stream, launch_rmsnorm(ACACHE_BF16, x, w->mlp_norm, y, M, d, dims->rms_eps, stream));
  } else {
    g.P = part;
    LAUNCH_T(ACACHE_K_GEMM_O, stream, launch_gemm_bf16(EPI_PARTIAL, g, stream));
    LAUNCH_T(ACACHE_K_RESIDUAL, stream,
             launch_reduce_residual(x, part, g.splits, M, d, w->mlp_norm, y, dims->rms_eps, stream));
  }
  GemmParams u = {};
  u.X = y;
  u.W = w->w_gate_up;
  u.M = M;
  u.N = 2 * F;
  u.K = d;
  u.splits = 1;
  u.C = hb;
  u.ldc = F;
  u.sk_ws = part;
  LAUNCH_T(ACACHE_K_GEMM_GATE_UP, stream, launch_gemm_bf16(EPI_SWIGLU, u, stream));
  GemmParams dn = {};
  dn.X = hb;
  dn.W = w->w_down;
  dn.M = M;
  dn.N = d;
  dn.K = F;
  dn.splits = gemm_bf16_splits(M, d, F);
  if (dn.splits == 1) {
    dn.C = x;
    dn.ldc = d;
    dn.sk_ws = part;
    LAUNCH_T(ACACHE_K_GEMM_DOWN, stream, launch_gemm_bf16(EPI_ACCUM, dn, stream));
  } else {
    dn.P = part;
    LAUNCH_T(ACACHE_K_GEMM_DOWN, stream, launch_gemm_bf16(EPI_PARTIAL, dn, stream));
    LAUNCH_T(ACACHE_K_RESIDUAL, stream,
             launch_reduce_residual(x, part, dn.splits, M, d, nullptr, nullptr, dims->rms_eps, stream));
  }
  return ACACHE_OK;
}

acache_status acache_layer_recompute(const acache_dims* dims, const acache_layer_weights* w,
                                     const acache_ragged* rg, void* x, const int32_t* pos,
                                     const int32_t* write_slots, const int32_t* read_slots,
                                     void* k_pool, void* v_pool, int64_t pool_ld, int64_t n_slots,
                                     const acache_score_args* score, void* ws, size_t ws_bytes,
                                     hipStream_t stream) {
  acache_status st = check_layer_dims(dims);
  if (st != ACACHE_OK) return st;
  Ragged r;
  st = make_ragged(rg, r);
  if (st != ACACHE_OK) return st;
  const int M = r.cu_rows[r.batch];
  if (M == 0) return ACACHE_OK;
  CHECK(w && x && pos && write_slots && read_slots && k_pool && v_pool, ACACHE_ERR_NULL);
  CHECK(w->attn_norm && w->w_qkv && w->w_o && w->mlp_norm && w->w_gate_up && w->w_down, ACACHE_ERR_NULL);
  const int d = dims->d_model, H = dims->n_heads, Hkv = dims->n_kv_heads, dh = dims->head_dim,
            F = dims->d_ff;
  const int hq = H * dh, hkv = Hkv * dh, nqkv = (H + 2 * Hkv) * dh;
  CHECK(pool_ld >= hkv && n_slots > 0, ACACHE_ERR_SHAPE);
  CHECK(n_slots * pool_ld < ((int64_t)1 << 31), ACACHE_ERR_UNSUPPORTED);  // 32-bit element offsets
  // the projections address their operands with 32-bit element offsets
  CHECK((int64_t)M * std::max({d, hq, F}) < ((int64_t)1 << 31), ACACHE_ERR_UNSUPPORTED);
  CHECK((int64_t)std::max({nqkv, 2 * F, d}) * std::max({d, hq, F}) < ((int64_t)1 << 31), ACACHE_ERR_UNSUPPORTED);
  const int64_t es = (int64_t)elem_size(dims->dtype);
  CHECK(aligned16(x) && aligned16(k_pool) && aligned16(v_pool) && (pool_ld * es) % 16 == 0, ACACHE_ERR_ALIGN);
  CHECK(aligned16(w->attn_norm) && aligned16(w->w_qkv) && aligned16(w->w_o) && aligned16(w->mlp_norm) &&
            aligned16(w->w_gate_up) && aligned16(w->w_down),
        ACACHE_ERR_ALIGN);
  int L = 0;
  if (score) {
    L = score->affix_len;
    CHECK(L >= 0 && L <= 65536, ACACHE_ERR_SHAPE);
    CHECK(score->norm == ACACHE_NORM_AFFIX || score->norm == ACACHE_NORM_FULL, ACACHE_ERR_UNSUPPORTED);
    st = check_cu(score->cu_q, r.batch);
    if (st != ACACHE_OK) return st;
    CHECK(score->cu_q[r.batch] <= M, ACACHE_ERR_SHAPE);
    if (L > 0 && score->cu_q[r.batch] > 0) CHECK(score->q_rows && score->affix_slots && score->scores, ACACHE_ERR_NULL);
  }
  const WsPlan p = plan_ws(dims, M, r.batch, L);
  CHECK(ws && ws_bytes >= p.total && aligned16(ws), ACACHE_ERR_WORKSPACE);
  void* y = at<char>(ws, p.y);
  void* q = at<char>(ws, p.q);
  void* o = at<char>(ws, p.o);
  void* hb = at<char>(ws, p.h);
  const bool probe = score && L > 0 && score->cu_q[r.batch] > 0;
  float* lse = (probe && score->norm == ACACHE_NORM_FULL) ? at<float>(ws, p.lse) : nullptr;
  // under the affix normaliser the attention may take the rows' log-sum-exp
  // over the affix keys for the score, where the caller promises every
  // request reads them in order from key index affix_key_begin
  float* lse_aff = nullptr;
  if (probe && score->norm == ACACHE_NORM_AFFIX && dims->dtype == ACACHE_BF16 && score->affix_keys_known &&
      score->affix_key_begin >= 0) {
    bool fits = true;
    for (int b = 0; b < r.batch; ++b)
      fits = fits && (int64_t)r.cu_keys[b + 1] - r.cu_keys[b] >= (int64_t)score->affix_key_begin + L;
    if (fits) lse_aff = at<float>(ws, p.lse_aff);
  }
  bool aff_done = false;

  LAUNCH_T(ACACHE_K_RMSNORM, stream, launch_rmsnorm(dims->dtype, x, w->attn_norm, y, M, d, dims->rms_eps, stream));
  if (dims->dtype == ACACHE_BF16) {
    st = run_qkv_bf16(dims, w, M, y, q, pos, write_slots, k_pool, v_pool, pool_ld, n_slots, at<float>(ws, p.part),
                      at<float>(ws, p.rope), stream);
    if (st != ACACHE_OK) return st;
    // the part region is idle between the QKV fixup and the O projection
    LAUNCH_T(ACACHE_K_ATTENTION, stream, launch_attention_bf16(r, H, Hkv, q, read_slots, k_pool, v_pool, pool_ld, n_slots, o, lse,
                                                                at<float>(ws, p.part), p.part_bytes, stream, lse_aff,
                                                                lse_aff ? score->affix_key_begin : 0, L, &aff_done));
  } else {
    float* qkv = at<float>(ws, p.qkv);
    LAUNCH_T(ACACHE_K_GEMM_QKV, stream, launch_gemm_f32((const float*)y, (const float*)w->w_qkv, qkv, nqkv, M, nqkv, d, 0, stream));
    LAUNCH(launch_rope_scatter_f32(qkv, M, H, Hkv, dh, pos, dims->rope_base, (float*)q, write_slots,
                                   (float*)k_pool, (float*)v_pool, pool_ld, n_slots, stream));
    LAUNCH_T(ACACHE_K_ATTENTION, stream, launch_attention_f32(r, H, Hkv, dh, (const float*)q, read_slots, (const float*)k_pool,
                                (const float*)v_pool, pool_ld, n_slots, (float*)o, lse, stream));
  }
  if (probe) {
    st = run_score(dims, r.batch, score->cu_q, q, hq, M, score->q_rows, k_pool, pool_ld, n_slots,
                   score->affix_slots, L, score->norm, lse, score->scores, at<float>(ws, p.lse_aff),
                   at<float>(ws, p.colsum), p.colsum_bytes, score->init, stream, aff_done ? lse_aff : nullptr);
    if (st != ACACHE_OK) return st;
  }
  if (dims->dtype == ACACHE_BF16) {
    st = run_out_mlp_bf16(dims, w, M, x, y, o, hb, at<float>(ws, p.part), stream);
    if (st != ACACHE_OK) return st;
  } else {
    float* gu = at<float>(ws, p.gu);
    LAUNCH_T(ACACHE_K_GEMM_O, stream, launch_gemm_f32((const float*)o, (const float*)w->w_o, (float*)x, d, M, d, hq, 1, stream));
    LAUNCH(launch_rmsnorm(ACACHE_F32, x, w->mlp_norm, y, M, d, dims->rms_eps, stream));
    LAUNCH_T(ACACHE_K_GEMM_GATE_UP, stream, launch_gemm_f32((const float*)y, (const float*)w->w_gate_up, gu, 2 * F, M, 2 * F, d, 0, stream));
    LAUNCH(launch_swiglu_f32(gu, M, F, (float*)hb, stream));
    LAUNCH_T(ACACHE_K_GEMM_DOWN, stream, launch_gemm_f32((const float*)hb, (const float*)w->w_down, (float*)x, d, M, d, F, 1, stream));
  }
  return ACACHE_OK;
}

acache_status acache_layer_score(const acache_dims* dims, const acache_layer_weights* w, const acache_ragged* rg,
                                 const void* x, const int32_t* pos, const int32_t* write_slots,
                                 const int32_t* read_slots, void* k_pool, void* v_pool, int64_t pool_ld,
                                 int64_t n_slots, const acache_score_args* score, void* ws, size_t ws_bytes,
                                 hipStream_t stream) {
  acache_status st = check_layer_dims(dims);
  if (st != ACACHE_OK) return st;
  CHECK(score, ACACHE_ERR_NULL);
  Ragged r;
  st = make_ragged(rg, r);
  if (st != ACACHE_OK) return st;
  const int M = r.cu_rows[r.batch];
  const int L = score->affix_len;
  CHECK(L >= 0 && L <= 65536, ACACHE_ERR_SHAPE);
  CHECK(score->norm == ACACHE_NORM_AFFIX || score->norm == ACACHE_NORM_FULL, ACACHE_ERR_UNSUPPORTED);
  st = check_cu(score->cu_q, r.batch);
  if (st != ACACHE_OK) return st;
  CHECK(score->cu_q[r.batch] <= M, ACACHE_ERR_SHAPE);
  const int Mq = score->cu_q[r.batch];
  if (M == 0 || L == 0 || Mq == 0) return ACACHE_OK;  // nothing to add
  CHECK(score->q_rows && score->affix_slots && score->scores, ACACHE_ERR_NULL);
  const bool full = score->norm == ACACHE_NORM_FULL;
  CHECK(w && x && pos && k_pool, ACACHE_ERR_NULL);
  CHECK(w->attn_norm && w->w_qkv, ACACHE_ERR_NULL);
  // the full softmax's normaliser needs every row's keys and the attention
  CHECK(!full || (write_slots && read_slots && v_pool), ACACHE_ERR_NULL);
  const int d = dims->d_model, H = dims->n_heads, Hkv = dims->n_kv_heads, dh = dims->head_dim;
  const int hq = H * dh, hkv = Hkv * dh, nqkv = (H + 2 * Hkv) * dh;
  CHECK(pool_ld >= hkv && n_slots > 0, ACACHE_ERR_SHAPE);
  CHECK(n_slots * pool_ld < ((int64_t)1 << 31), ACACHE_ERR_UNSUPPORTED);
  CHECK((int64_t)M * std::max(d, hq) < ((int64_t)1 << 31), ACACHE_ERR_UNSUPPORTED);
  CHECK((int64_t)nqkv * std::max(d, hq) < ((int64_t)1 << 31), ACACHE_ERR_UNSUPPORTED);
  const int64_t es = (int64_t)elem_size(dims->dtype);
  CHECK(aligned16(x) && aligned16(k_pool) && (pool_ld * es) % 16 == 0, ACACHE_ERR_ALIGN);
  CHECK(!full || aligned16(v_pool), ACACHE_ERR_ALIGN);
  CHECK(aligned16(w->attn_norm) && aligned16(w->w_qkv), ACACHE_ERR_ALIGN);
  const WsPlan p = plan_ws(dims, M, r.batch, L);
  CHECK(ws && ws_bytes >= p.total && aligned16(ws), ACACHE_ERR_WORKSPACE);
  void* y = at<char>(ws, p.y);
  void* q = at<char>(ws, p.q);
  float* lse = full ? at<float>(ws, p.lse) : nullptr;

  if (dims->dtype == ACACHE_BF16 && !full) {
    // the masked rows only: gather, normalise, project to queries (split-K
    // over the whole chip), then sum the splits and rotate
    CHECK(dims->d_ff >= d, ACACHE_ERR_UNSUPPORTED);  // the gathered rows sit in the MLP region
    if (rmsnorm_rows_ok(x, w->attn_norm, y, d)) {
      LAUNCH_T(ACACHE_K_RMSNORM, stream,
               launch_rmsnorm_rows(x, M, score->q_rows, w->attn_norm, y, Mq, d, dims->rms_eps, stream));
    } else {
      void* xq = at<char>(ws, p.h);
      LAUNCH_T(ACACHE_K_GATHER, stream, launch_gather_rows(x, (int64_t)d * 2, M, score->q_rows, nullptr, 0, Mq,
                                                           d * 2, xq, (int64_t)d * 2, stream));
      LAUNCH_T(ACACHE_K_RMSNORM, stream, launch_rmsnorm(ACACHE_BF16, xq, w->attn_norm, y, Mq, d, dims->rms_eps, stream));
    }
    GemmParams g = {};
    g.X = y;
    g.W = w->w_qkv;  // the query rows come first
    g.M = Mq;
    g.N = hq;
    g.K = d;
    g.splits = gemm_bf16_splits(Mq, hq, d);
    g.P = at<float>(ws, p.part);
    CHECK((size_t)g.splits * Mq * hq * sizeof(float) <= p.part_bytes, ACACHE_ERR_WORKSPACE);
    LAUNCH_T(ACACHE_K_GEMM_QKV, stream, launch_gemm_bf16(EPI_PARTIAL, g, stream));
    LAUNCH_T(ACACHE_K_RESIDUAL, stream, launch_q_rotary_reduce(g.P, g.splits, Mq, H, score->q_rows, pos,
                                                               dims->rope_base, q, M, stream));
  } else {
    LAUNCH_T(ACACHE_K_RMSNORM, stream, launch_rmsnorm(dims->dtype, x, w->attn_norm, y, M, d, dims->rms_eps, stream));
    if (dims->dtype == ACACHE_BF16) {
      st = run_qkv_bf16(dims, w, M, y, q, pos, write_slots, k_pool, v_pool, pool_ld, n_slots, at<float>(ws, p.part),
                        at<float>(ws, p.rope), stream);
      if (st != ACACHE_OK) return st;
      LAUNCH_T(ACACHE_K_ATTENTION, stream, launch_attention_bf16(r, H, Hkv, q, read_slots, k_pool, v_pool, pool_ld,
                                                                  n_slots, at<char>(ws, p.o), lse,
                                                                  at<float>(ws, p.part), p.part_bytes, stream));
    } else {
      float* qkv = at<float>(ws, p.qkv);
      LAUNCH_T(ACACHE_K_GEMM_QKV, stream, launch_gemm_f32((const float*)y, (const float*)w->w_qkv, qkv, nqkv, M, nqkv, d, 0, stream));
      // the pools are written only when the attention reads them (with
      // n_slots 0 no slot is valid and nothing is stored; pos then stands
      // in for the slot list, which the affix-only reading does not need)
      LAUNCH(launch_rope_scatter_f32(qkv, M, H, Hkv, dh, pos, dims->rope_base, (float*)q, full ? write_slots : pos,
                                     (float*)k_pool, (float*)v_pool, pool_ld, full ? n_slots : 0, stream));
      if (full)
        LAUNCH_T(ACACHE_K_ATTENTION, stream, launch_attention_f32(r, H, Hkv, dh, (const float*)q, read_slots,
                                                                   (const float*)k_pool, (const float*)v_pool, pool_ld,
                                                                   n_slots, at<float>(ws, p.o), lse, stream));
    }
  }
  return run_score(dims, r.batch, score->cu_q, q, hq, M, score->q_rows, k_pool, pool_ld, n_slots, score->affix_slots, L,
                   score->norm, lse, score->scores, at<float>(ws, p.lse_aff), at<float>(ws, p.colsum),
                   p.colsum_bytes, score->init, stream);
}

acache_status acache_layer_decode(const acache_dims* dims, const acache_layer_weights* w, int32_t batch,
                                  int32_t rows_per_request, void* x, const int32_t* pos, const int32_t* write_slots,
                                  const int32_t* affix_slots, int32_t affix_len, const int32_t* anchors, int32_t k,
                                  const int32_t* private_slots, int32_t private_len, void* k_pool, void* v_pool,
                                  int64_t pool_ld, int64_t n_slots, void* ws, size_t ws_bytes, hipStream_t stream) {
  acache_status st = check_layer_dims(dims);
  if (st != ACACHE_OK) return st;
  CHECK(dims->dtype == ACACHE_BF16, ACACHE_ERR_UNSUPPORTED);
  CHECK(batch >= 0 && batch <= 64 && rows_per_request >= 0 && affix_len >= 0 && affix_len <= 65536, ACACHE_ERR_SHAPE);
  CHECK(k >= 0 && k <= affix_len && private_len >= 0, ACACHE_ERR_SHAPE);
  const int64_t M64 = (int64_t)batch * rows_per_request;
  CHECK(M64 < ((int64_t)1 << 31), ACACHE_ERR_SHAPE);
  const int M = (int)M64;
  if (M == 0) return ACACHE_OK;
  CHECK(private_len > 0 || affix_len > k, ACACHE_ERR_SHAPE);  // every request has keys
  CHECK(w && x && pos && write_slots && k_pool && v_pool, ACACHE_ERR_NULL);
  CHECK(w->attn_norm && w->w_qkv && w->w_o && w->mlp_norm && w->w_gate_up && w->w_down, ACACHE_ERR_NULL);
  CHECK(affix_len == k || affix_slots, ACACHE_ERR_NULL);
  CHECK(k == 0 || affix_len == k || anchors, ACACHE_ERR_NULL);
  CHECK(private_len == 0 || private_slots, ACACHE_ERR_NULL);
  const int d = dims->d_model, H = dims->n_heads, Hkv = dims->n_kv_heads, dh = dims->head_dim, F = dims->d_ff;
  const int hq = H * dh, hkv = Hkv * dh, nqkv = (H + 2 * Hkv) * dh;
  CHECK(pool_ld >= hkv && n_slots > 0, ACACHE_ERR_SHAPE);
  CHECK(n_slots * pool_ld < ((int64_t)1 << 31), ACACHE_ERR_UNSUPPORTED);
  CHECK((int64_t)M * std::max({d, hq, F}) < ((int64_t)1 << 31), ACACHE_ERR_UNSUPPORTED);
  CHECK((int64_t)std::max({nqkv, 2 * F, d}) * std::max({d, hq, F}) < ((int64_t)1 << 31), ACACHE_ERR_UNSUPPORTED);
  CHECK(aligned16(x) && aligned16(k_pool) && aligned16(v_pool) && (pool_ld * 2) % 16 == 0, ACACHE_ERR_ALIGN);
  CHECK(aligned16(w->attn_norm) && aligned16(w->w_qkv) && aligned16(w->w_o) && aligned16(w->mlp_norm) &&
            aligned16(w->w_gate_up) && aligned16(w->w_down),
        ACACHE_ERR_ALIGN);
  const WsPlan p = plan_ws(dims, M, batch, affix_len);
  CHECK(ws && ws_bytes >= p.total && aligned16(ws), ACACHE_ERR_WORKSPACE);
  // the anchor masks live in the scoring region, which a decode step does not use
  const size_t mask_bytes = (size_t)batch * ((affix_len + 63) / 64) * sizeof(uint64_t);
  CHECK(mask_bytes <= (size_t)batch * H * std::max(affix_len, 1) * sizeof(float), ACACHE_ERR_WORKSPACE);
  CHECK((size_t)M * H * (dh * 4 + 8) * 2 <= p.part_bytes, ACACHE_ERR_WORKSPACE);
  void* y = at<char>(ws, p.y);
  void* q = at<char>(ws, p.q);
  void* o = at<char>(ws, p.o);
  void* hb = at<char>(ws, p.h);
  float* part = at<float>(ws, p.part);

  LAUNCH_T(ACACHE_K_RMSNORM, stream, launch_rmsnorm(ACACHE_BF16, x, w->attn_norm, y, M, d, dims->rms_eps, stream));
  st = run_qkv_bf16(dims, w, M, y, q, pos, write_slots, k_pool, v_pool, pool_ld, n_slots, part, at<float>(ws, p.rope),
                    stream);
  if (st != ACACHE_OK) return st;
  LAUNCH_T(ACACHE_K_ATTENTION, stream,
           launch_attention_decode_bf16(batch, rows_per_request, H, Hkv, q, affix_slots, affix_len, anchors, k,
                                        private_slots, private_len, k_pool, v_pool, pool_ld, n_slots, o,
                                        at<uint64_t>(ws, p.colsum), part, p.part_bytes, stream));
  return run_out_mlp_bf16(dims, w, M, x, y, o, hb, part, stream);
}

}  // extern "C"
