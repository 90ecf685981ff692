// Row-level kernels: gather of recomputed rows, K/V scatter to pool slots,
// the write/read slot maps, RMSNorm, split-K reduction with residual add and
// RMSNorm, and the per-head reduction of probe scores.  All are HBM-bound
// row copies or row reductions: 16-byte vector accesses, one row per
// workgroup or grid-stride over 16-byte chunks.
#include "device.h"
#include "internal.h"

namespace acache {

namespace {

typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4;

// ---------------------------------------------------------------- gather (Section 4.3)
__global__ __launch_bounds__(256) void gather_rows_kernel(const char* __restrict__ src, int64_t src_ld,
                                                          int64_t src_rows, const int32_t* __restrict__ idx,
                                                          const int32_t* __restrict__ remap, int64_t remap_len,
                                                          int n, int chunks, char* __restrict__ dst,
                                                          int64_t dst_ld) {
  const int64_t total = (int64_t)n * chunks;
  for (int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; c < total;
       c += (int64_t)gridDim.x * blockDim.x) {
    const int i = (int)(c / chunks);
    const int ch = (int)(c - (int64_t)i * chunks);
    int64_t r = idx[i];
    bool ok = true;
    if (remap) {
      ok = r >= 0 && r < remap_len;
      r = ok ? remap[r] : 0;
    }
    ok = ok && r >= 0 && r < src_rows;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (ok) v = *reinterpret_cast<const u32x4*>(src + r * src_ld + (int64_t)ch * 16);
    *reinterpret_cast<u32x4*>(dst + (int64_t)i * dst_ld + (int64_t)ch * 16) = v;
  }
}

// ---------------------------------------------------------------- scatter (Appendix C.1 store)
__global__ __launch_bounds__(256) void kv_scatter_kernel(const char* __restrict__ ks, const char* __restrict__ vs,
                                                         int64_t src_ld, int n, const int32_t* __restrict__ slots,
                                                         char* __restrict__ kp, char* __restrict__ vp,
                                                         int64_t pool_ld, int64_t n_slots, int chunks) {
  const int64_t total = (int64_t)n * chunks;
  for (int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; c < total;
       c += (int64_t)gridDim.x * blockDim.x) {
    const int i = (int)(c / chunks);
    const int ch = (int)(c - (int64_t)i * chunks);
    const int64_t slot = slots[i];
    if (slot < 0 || slot >= n_slots) continue;
    const int64_t so = (int64_t)i * src_ld + (int64_t)ch * 16;
    const int64_t po = slot * pool_ld + (int64_t)ch * 16;
    *reinterpret_cast<u32x4*>(kp + po) = *reinterpret_cast<const u32x4*>(ks + so);
    *reinterpret_cast<u32x4*>(vp + po) = *reinterpret_cast<const u32x4*>(vs + so);
  }
}

// ---------------------------------------------------------------- maps (Section 4.1)
// Slot of index i in a block table (block_size consecutive slots per block);
// -1 where the slot does not fit in int32.
__device__ __forceinline__ int32_t paged_slot(const int32_t* __restrict__ table, int bs, int i) {
  const int64_t s = (int64_t)table[i / bs] * bs + (i % bs);
  return (s >= 0 && s <= INT32_MAX) ? (int32_t)s : -1;
}

// With pg.block_size > 0 the slots come from the paging plan's block tables;
// otherwise from the layout's shared_base / private_base / private_stride.
__global__ __launch_bounds__(256) void build_maps_kernel(acache_layout lay, acache_paging pg, int batch,
                                                         const int32_t* __restrict__ anchors, int k,
                                                         int32_t* __restrict__ row_pos,
                                                         int32_t* __restrict__ row_src,
                                                         int32_t* __restrict__ wslots,
                                                         int32_t* __restrict__ rslots,
                                                         int32_t* __restrict__ q_rows) {
  const int S = lay.seq_len, ab = lay.affix_begin, L = lay.affix_len;
  const int ae = ab + L;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= (int64_t)batch * S) return;
  const int b = (int)(t / S);
  const int p = (int)(t - (int64_t)b * S);
  const int R = k + S - L;
  bool rec = true;
  int rank;
  if (p < ab) {
    rank = p;
  } else if (p >= ae) {
    rank = ab + k + (p - ae);
  } else {
    // lower bound of the affix-local index among the request's anchors
    const int a = p - ab;
    const int32_t* an = anchors + (int64_t)b * k;
    int lo = 0, hi = k;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (an[mid] < a) lo = mid + 1; else hi = mid;
    }
    rec = lo < k && an[lo] == a;
    rank = ab + lo;
  }
  int32_t slot;
  if (rec) {
    slot = pg.block_size > 0
               ? paged_slot(pg.private_blocks + (int64_t)b * pg.blocks_per_request, pg.block_size, rank)
               : lay.private_base + b * lay.private_stride + rank;
    const int64_t row = (int64_t)b * R + rank;
    row_pos[row] = p;
    row_src[row] = b * S + p;
    wslots[row] = slot;
    if (q_rows && p >= lay.mask_begin && p < lay.mask_begin + lay.mask_len)
      q_rows[(int64_t)b * lay.mask_len + (p - lay.mask_begin)] = (int32_t)row;
  } else {
    slot = pg.block_size > 0 ? paged_slot(pg.shared_blocks, pg.block_size, p - ab) : lay.shared_base + (p - ab);
  }
  // key index of position p: p, or with the affix first p - ab inside the
  // affix, L + p before it and p after it
  const int key = lay.key_order == 0 ? p : (p >= ab && p < ae) ? p - ab : p < ab ? L + p : p;
  rslots[(int64_t)b * S + key] = slot;
}

// ---------------------------------------------------------------- RMSNorm
template <typename T>
__global__ __launch_bounds__(256) void rmsnorm_kernel(const T* __restrict__ x, const T* __restrict__ g,
                                                      T* __restrict__ y, int d, float eps) {
  const int64_t row = blockIdx.x;
  const T* xr = x + row * d;
  T* yr = y + row * d;
  __shared__ float red[4];
  float ss = 0.f;
  for (int i = threadIdx.x; i < d; i += 256) {
    const float v = to_f32(xr[i]);
    ss += v * v;
  }
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float tot = red[0] + red[1] + red[2] + red[3];
  const float inv = rsqrtf(tot / (float)d + eps);
  for (int i = threadIdx.x; i < d; i += 256) yr[i] = from_f32<T>(to_f32(xr[i]) * inv * to_f32(g[i]));
}

// bf16 rows with d % 8 == 0, d <= 8192 and 16-byte aligned rows: 16-byte
// loads, the row kept in registers between the sum of squares and the
// scaling, and the gain loaded before the reduction.  Same arithmetic as
// rmsnorm_kernel (x * inv * g per element).
// With rows, output row i normalises x[rows[i]] (the gather fused in; a row
// index outside [0, n_src) gives a zero row, as the gather does).
__global__ __launch_bounds__(256) void rmsnorm_vec_kernel(const bf16* __restrict__ x, const bf16* __restrict__ g,
                                                          bf16* __restrict__ y, int d, float eps,
                                                          const int32_t* __restrict__ rows, int64_t n_src) {
  const int64_t row = blockIdx.x;
  int64_t src = row;
  bool ok = true;
  if (rows != nullptr) {
    src = rows[row];
    ok = src >= 0 && src < n_src;
    if (!ok) src = 0;
  }
  const int nch = d >> 3;
  bf16x8 xv[4], gv[4];
  float ss = 0.f;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int ch = threadIdx.x + c * 256;
    if (ch < nch) {
      xv[c] = *reinterpret_cast<const bf16x8*>(x + src * d + (int64_t)ch * 8);
      gv[c] = *reinterpret_cast<const bf16x8*>(g + (int64_t)ch * 8);
      if (!ok) xv[c] = bf16x8{};
    }
  }
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    if (threadIdx.x + c * 256 < nch) {
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float v = (float)xv[c][j];
        ss += v * v;
      }
    }
  }
  __shared__ float red[4];
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float inv = rsqrtf((red[0] + red[1] + red[2] + red[3]) / (float)d + eps);
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int ch = threadIdx.x + c * 256;
    if (ch < nch) {
      bf16x8 o;
#pragma unroll
      for (int j = 0; j < 8; ++j) o[j] = (bf16)((float)xv[c][j] * inv * (float)gv[c][j]);
      *reinterpret_cast<bf16x8*>(y + row * d + (int64_t)ch * 8) = o;
    }
  }
}

// ---------------------------------------------------------------- split-K reduce + rotary (queries only)
// The probe's last layer projects only the masked rows' queries, as fp32
// split-K partials [splits][n][H * 128].  One thread per (row, head, 4 of
// the 64 rotary pairs): the splits are summed in order, the pairs (d, d + 64)
// are rotated by the row's position exactly as the Q/K/V projection's
// epilogue does (fp64 angle, rotary_sincos), and the row is written to
// q[rows[i]] (rows outside [0, q_n_rows) are skipped).
__global__ __launch_bounds__(256) void q_rotary_reduce_kernel(const float* __restrict__ part, int splits, int n,
                                                              int H, const int32_t* __restrict__ rows,
                                                              const int32_t* __restrict__ pos, float rope_base,
                                                              bf16* __restrict__ q, int64_t q_n_rows) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= (int64_t)n * H * 16) return;
  const int i = (int)(t / (H * 16));
  const int rem = (int)(t - (int64_t)i * H * 16);
  const int h = rem >> 4, d0 = (rem & 15) * 4;
  const int64_t hq = (int64_t)H * 128;
  const int64_t r = rows[i];
  if (r < 0 || r >= q_n_rows) return;
  float lo[4] = {0.f, 0.f, 0.f, 0.f}, hi[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
  for (int sp = 0; sp < splits; ++sp) {
    const float* pp = part + ((int64_t)sp * n + i) * hq + h * 128 + d0;
    const f32x4 a = *reinterpret_cast<const f32x4*>(pp);
    const f32x4 b = *reinterpret_cast<const f32x4*>(pp + 64);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      lo[j] += a[j];
      hi[j] += b[j];
    }
  }
  const double ang_pos = (double)pos[r];
  const double l2b = log2((double)rope_base);
  bf16x4 olo, ohi;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int d = d0 + j;
    float sn, cs;
    rotary_sincos(ang_pos * exp2(-(2.0 * d / 128.0) * l2b), &sn, &cs);
    olo[j] = (bf16)(lo[j] * cs - hi[j] * sn);
    ohi[j] = (bf16)(hi[j] * cs + lo[j] * sn);
  }
  bf16* dst = q + r * hq + h * 128 + d0;
  *reinterpret_cast<bf16x4*>(dst) = olo;
  *reinterpret_cast<bf16x4*>(dst + 64) = ohi;
}

// ---------------------------------------------------------------- split-K reduce + residual (+ RMSNorm)
// One workgroup per row; each thread keeps NC chunks of 8 columns in
// registers between the residual sum and the normalisation (d <= 8192).
// Chunk c of thread t is column chunk t + 256 c; the loads are issued for
// all NC chunks of a split (clamped to the last chunk, results of absent
// chunks unused) so that they are in flight together.  Each element is
// x + p_0 + p_1 + ... in split order.
template <int NC>
__global__ __launch_bounds__(256) void reduce_residual_kernel(bf16* __restrict__ x, const float* __restrict__ part,
                                                              int splits, int M, int d,
                                                              const bf16* __restrict__ g,
                                                              bf16* __restrict__ y, float eps) {
  const int64_t row = blockIdx.x;
  const int nch = d >> 3;
  int64_t off[NC];
  bool ok[NC];
  float v[NC][8];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int ch = threadIdx.x + c * 256;
    ok[c] = ch < nch;
    off[c] = row * d + (int64_t)min(ch, nch - 1) * 8;
    const bf16x8 xv = *reinterpret_cast<const bf16x8*>(x + off[c]);
#pragma unroll
    for (int j = 0; j < 8; ++j) v[c][j] = (float)xv[j];
  }
#pragma unroll 2
  for (int sp = 0; sp < splits; ++sp) {
    f32x4 a[NC], b[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const float* pp = part + (int64_t)sp * M * d + off[c];
      a[c] = *reinterpret_cast<const f32x4*>(pp);
      b[c] = *reinterpret_cast<const f32x4*>(pp + 4);
    }
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        v[c][j] += a[c][j];
        v[c][4 + j] += b[c][j];
      }
  }
  float ss = 0.f;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    bf16x8 o;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      o[j] = (bf16)v[c][j];
      v[c][j] = (float)o[j];
    }
    if (ok[c]) {
#pragma unroll
      for (int j = 0; j < 8; ++j) ss += v[c][j] * v[c][j];
      *reinterpret_cast<bf16x8*>(x + off[c]) = o;
    }
  }
  if (!y) return;
  __shared__ float red[4];
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float inv = rsqrtf((red[0] + red[1] + red[2] + red[3]) / (float)d + eps);
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    if (ok[c]) {
      const int ch = threadIdx.x + c * 256;
      const bf16x8 gv = *reinterpret_cast<const bf16x8*>(g + (int64_t)ch * 8);
      bf16x8 o;
#pragma unroll
      for (int j = 0; j < 8; ++j) o[j] = (bf16)(v[c][j] * inv * (float)gv[j]);
      *reinterpret_cast<bf16x8*>(y + off[c]) = o;
    }
  }
}

// ---------------------------------------------------------------- probe-score head reduction (Eq. 5)
// scores[b][j] (+)= sum over the request's R partial rows part[b][r][j], in
// a fixed order: 8 chunks of consecutive rows summed by 8 threads (rows in
// ascending order), then the 8 chunk sums in chunk order.  Workgroup: 32
// keys x 8 chunks.
__global__ __launch_bounds__(256) void head_reduce_kernel(const float* __restrict__ part, int batch, int R,
                                                          int L, float* __restrict__ scores, int init) {
  __shared__ float cs[8][33];
  const int kx = threadIdx.x & 31, c = threadIdx.x >> 5;
  const int64_t t = (int64_t)blockIdx.x * 32 + kx;
  const bool ok = t < (int64_t)batch * L;
  const int b = ok ? (int)(t / L) : 0;
  const int j = ok ? (int)(t - (int64_t)b * L) : 0;
  const int r0 = c * R / 8, r1 = (c + 1) * R / 8;
  const float* p = part + (int64_t)b * R * L + j;
  float s = 0.f;
  if (ok) {
#pragma unroll 4
    for (int r = r0; r < r1; ++r) s += p[(int64_t)r * L];
  }
  cs[c][kx] = s;
  __syncthreads();
  if (c == 0 && ok) {
    float tot = cs[0][kx];
#pragma unroll
    for (int i = 1; i < 8; ++i) tot += cs[i][kx];
    scores[t] = init ? tot : scores[t] + tot;
  }
}

inline int grid_for(int64_t work, int per_block = 256, int cap = 65535) {
  int64_t g = (work + per_block - 1) / per_block;
  if (g < 1) g = 1;
  return (int)(g > cap ? cap : g);
}


// ---------------------------------------------------------------- greedy commit
// One workgroup per row: the index of the largest element by order_key (NaN
// lowest, -0 == +0), the lowest index among equal keys.  out[row] = index and,
// with commit_pos, ids[commit_pos[row]] = index (an out-of-range position is
// skipped).
__device__ __forceinline__ void argmax_take(uint32_t key, int idx, uint32_t& bk, int& bi) {
  if (key > bk || (key == bk && idx < bi)) {
    bk = key;
    bi = idx;
  }
}
__device__ __forceinline__ uint32_t elem_bits(bf16 v) { return (uint32_t)__builtin_bit_cast(uint16_t, v) << 16; }
__device__ __forceinline__ uint32_t elem_bits(float v) { return __builtin_bit_cast(uint32_t, v); }

// Online softmax sum: (m, s) with s = sum exp(x - m) over the finite values
// seen (NaN and -inf add nothing); combining rescales the smaller maximum.
__device__ __forceinline__ void softmax_add(float x, float& m, float& s) {
  if (!(x > -INFINITY)) return;  // NaN or -inf
  if (x > m) {
    s = s * __expf(m - x) + 1.f;
    m = x;
  } else if (x == m) {
    s += 1.f;  // exact, also for an infinite maximum
  } else {
    s += __expf(x - m);
  }
}
__device__ __forceinline__ void softmax_merge(float m2, float s2, float& m, float& s) {
  if (s2 == 0.f) return;
  if (s != 0.f && m2 == m) {
    s += s2;
    return;
  }
  if (s == 0.f || m2 > m) {
    s = s2 + (s == 0.f ? 0.f : s * __expf(m - m2));
    m = m2;
  } else {
    s += s2 * __expf(m2 - m);
  }
}

template <typename T>
__global__ __launch_bounds__(256) void argmax_commit_kernel(const T* __restrict__ x, int64_t ld, int n, int vec,
                                                            int32_t* __restrict__ out, float* __restrict__ conf,
                                                            const int32_t* __restrict__ commit_pos,
                                                            int32_t* __restrict__ ids, int64_t ids_len) {
  constexpr int PER = 16 / sizeof(T);
  const int64_t row = blockIdx.x;
  const T* xr = x + row * ld;
  uint32_t bk = 0u;
  int bi = 0x7FFFFFFF;
  float sm = -INFINITY, ss = 0.f;
  int start = 0;
  if (vec) {
    const int chunks = n / PER;
    for (int c = threadIdx.x; c < chunks; c += 256) {
      const u32x4 raw = *reinterpret_cast<const u32x4*>(xr + (int64_t)c * PER);
      T v[PER];
      __builtin_memcpy(v, &raw, 16);
#pragma unroll
      for (int j = 0; j < PER; ++j) {
        argmax_take(order_key(elem_bits(v[j])), c * PER + j, bk, bi);
        if (conf) softmax_add(to_f32(v[j]), sm, ss);
      }
    }
    start = chunks * PER;
  }
  for (int i = start + threadIdx.x; i < n; i += 256) {
    argmax_take(order_key(elem_bits(xr[i])), i, bk, bi);
    if (conf) softmax_add(to_f32(xr[i]), sm, ss);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const uint32_t ok = __shfl_xor(bk, o);
    const int oi = __shfl_xor(bi, o);
    argmax_take(ok, oi, bk, bi);
    const float om = __shfl_xor(sm, o), os = __shfl_xor(ss, o);
    softmax_merge(om, os, sm, ss);
  }
  __shared__ uint32_t sk[4];
  __shared__ int si[4];
  __shared__ float smm[4], sss[4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) {
    sk[wave] = bk;
    si[wave] = bi;
    smm[wave] = sm;
    sss[wave] = ss;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
#pragma unroll
    for (int w = 1; w < 4; ++w) {
      argmax_take(sk[w], si[w], bk, bi);
      softmax_merge(smm[w], sss[w], sm, ss);
    }
    out[row] = bi;
    // probability of the largest finite logit (the argmax unless the row has +inf or only NaN)
    if (conf) conf[row] = ss > 0.f ? 1.f / ss : 0.f;
    if (commit_pos) {
      const int64_t p = commit_pos[row];
      if (p >= 0 && p < ids_len) ids[p] = bi;
    }
  }
}

// ---------------------------------------------------------------- shifted reuse
// Cached K is stored after rotation, so a span reused delta positions away
// is re-rotated in place of recomputation: each half-split pair (i, i + d_h/2)
// of every KV head turns by delta * theta_i (rotations compose).  One
// workgroup per row; each thread owns pairs, reading both halves before
// writing, so src and dst may be the same slot.
template <typename T>
__global__ __launch_bounds__(256) void rerotate_kernel(const T* __restrict__ src, int64_t src_ld,
                                                       const int32_t* __restrict__ src_slots, T* __restrict__ dst,
                                                       int64_t dst_ld, const int32_t* __restrict__ dst_slots,
                                                       const int32_t* __restrict__ delta, int64_t n_slots,
                                                       int heads, int dh, double log2_base) {
  const int row = blockIdx.x;
  const int64_t ss = src_slots[row], ds = dst_slots[row];
  if (ss < 0 || ss >= n_slots || ds < 0 || ds >= n_slots) return;
  const double dpos = (double)delta[row];
  const int half = dh >> 1;
  const T* sr = src + ss * src_ld;
  T* dr = dst + ds * dst_ld;
  for (int t = threadIdx.x; t < heads * half; t += blockDim.x) {
    const int h = t / half, i = t - h * half;
    const double inv_freq = exp2(-(2.0 * i / dh) * log2_base);
    float sn, cs;
    rotary_sincos(dpos * inv_freq, &sn, &cs);
    const float x1 = to_f32(sr[h * dh + i]), x2 = to_f32(sr[h * dh + i + half]);
    dr[h * dh + i] = from_f32<T>(x1 * cs - x2 * sn);
    dr[h * dh + i + half] = from_f32<T>(x2 * cs + x1 * sn);
  }
}

// ---------------------------------------------------------------- KV deviation
// The KV-deviation selector's score: for request b and affix token j,
// sum over the row's K and V elements of (fresh - shared)^2, fp32, one
// wavefront per (j, b), a fixed reduction order.
template <typename T>
__global__ __launch_bounds__(64) void kv_deviation_kernel(const T* __restrict__ kp, const T* __restrict__ vp,
                                                          int64_t pool_ld, int64_t n_slots,
                                                          const int32_t* __restrict__ fresh, int64_t fresh_ld,
                                                          const int32_t* __restrict__ stale, int L, int width,
                                                          float* __restrict__ scores) {
  constexpr int PER = 16 / sizeof(T);
  const int j = blockIdx.x, b = blockIdx.y, lane = threadIdx.x;
  const int64_t fs = fresh[(int64_t)b * fresh_ld + j], ss = stale[j];
  const bool ok = fs >= 0 && fs < n_slots && ss >= 0 && ss < n_slots;
  float acc = 0.f;
  if (ok) {
    const T* kf = kp + fs * pool_ld;
    const T* ks = kp + ss * pool_ld;
    const T* vf = vp + fs * pool_ld;
    const T* vs = vp + ss * pool_ld;
    for (int c = lane; c < width / PER; c += 64) {
      T a[PER], e[PER], f[PER], g[PER];
      __builtin_memcpy(a, kf + c * PER, 16);
      __builtin_memcpy(e, ks + c * PER, 16);
      __builtin_memcpy(f, vf + c * PER, 16);
      __builtin_memcpy(g, vs + c * PER, 16);
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        const float dk = to_f32(a[i]) - to_f32(e[i]), dv = to_f32(f[i]) - to_f32(g[i]);
        acc = fmaf(dk, dk, acc);
        acc = fmaf(dv, dv, acc);
      }
    }
  }
  acc = wave_sum(acc);
  if (lane == 0) scores[(int64_t)b * L + j] = ok ? acc : 0.f;
}

// ---------------------------------------------------------------- threshold commit
// One wavefront per request, over its block of `block` rows: every
// uncommitted row whose confidence reaches tau is committed; if none does,
// the single most confident uncommitted row (lowest row on equal
// confidence).  Committing writes the row's pick to ids[commit_pos[row]]
// and sets its flag; count[b] receives the number committed in this call.
__global__ __launch_bounds__(64) void threshold_commit_kernel(int block, const int32_t* __restrict__ pick,
                                                              const float* __restrict__ conf, float tau,
                                                              int32_t* __restrict__ committed,
                                                              const int32_t* __restrict__ commit_pos,
                                                              int32_t* __restrict__ ids, int64_t ids_len,
                                                              int32_t* __restrict__ count) {
  const int b = blockIdx.x, lane = threadIdx.x;
  int n_new = 0;
  // pass 1: threshold
  for (int r0 = 0; r0 < block; r0 += 64) {
    const int r = r0 + lane;
    const int64_t row = (int64_t)b * block + r;
    bool take = false;
    if (r < block && !committed[row]) take = conf[row] >= tau;
    if (take) {
      const int64_t p = commit_pos[row];
      if (p >= 0 && p < ids_len) ids[p] = pick[row];
      committed[row] = 1;
    }
    n_new += __popcll(__builtin_amdgcn_ballot_w64(take));
  }
  if (n_new == 0) {
    // pass 2: the most confident uncommitted row
    float best = -1.f;
    int best_r = 0x7FFFFFFF;
    for (int r0 = 0; r0 < block; r0 += 64) {
      const int r = r0 + lane;
      if (r < block && !committed[(int64_t)b * block + r]) {
        const float c = conf[(int64_t)b * block + r];
        const float ck = c == c ? c : -0.5f;  // NaN ranks below every confidence
        if (ck > best || (ck == best && r < best_r)) {
          best = ck;
          best_r = r;
        }
      }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float ob = __shfl_xor(best, o);
      const int orr = __shfl_xor(best_r, o);
      if (ob > best || (ob == best && orr < best_r)) {
        best = ob;
        best_r = orr;
      }
    }
    if (best_r < block) {
      if (lane == 0) {
        const int64_t row = (int64_t)b * block + best_r;
        const int64_t p = commit_pos[row];
        if (p >= 0 && p < ids_len) ids[p] = pick[row];
        committed[row] = 1;
      }
      n_new = 1;
    }
  }
  if (lane == 0) count[b] = n_new;
}
}  // namespace

hipError_t launch_gather_rows(const void* src, int64_t src_ld, int64_t src_rows, const int32_t* idx,
                              const int32_t* remap, int64_t remap_len, int n, int row_bytes,
                              void* dst, int64_t dst_ld, hipStream_t s) {
  const int chunks = row_bytes / 16;
  hipLaunchKernelGGL(gather_rows_kernel, dim3(grid_for((int64_t)n * chunks)), dim3(256), 0, s,
                     (const char*)src, src_ld, src_rows, idx, remap, remap_len, n, chunks,
                     (char*)dst, dst_ld);
  return hipGetLastError();
}

hipError_t launch_kv_scatter(const void* k_src, const void* v_src, int64_t src_ld_bytes, int n,
                             const int32_t* slots, void* k_pool, void* v_pool,
                             int64_t pool_ld_bytes, int64_t n_slots, int row_bytes, hipStream_t s) {
  const int chunks = row_bytes / 16;
  hipLaunchKernelGGL(kv_scatter_kernel, dim3(grid_for((int64_t)n * chunks)), dim3(256), 0, s,
                     (const char*)k_src, (const char*)v_src, src_ld_bytes, n, slots, (char*)k_pool,
                     (char*)v_pool, pool_ld_bytes, n_slots, chunks);
  return hipGetLastError();
}

hipError_t launch_build_maps(const acache_layout& lay, const acache_paging* paging, int batch,
                             const int32_t* anchors, int k, int32_t* row_pos, int32_t* row_src,
                             int32_t* write_slots, int32_t* read_slots, int32_t* q_rows, hipStream_t s) {
  const int64_t work = (int64_t)batch * lay.seq_len;
  acache_paging pg{};
  if (paging) pg = *paging;
  hipLaunchKernelGGL(build_maps_kernel, dim3((unsigned)((work + 255) / 256)), dim3(256), 0, s, lay, pg,
                     batch, anchors, k, row_pos, row_src, write_slots, read_slots, q_rows);
  return hipGetLastError();
}

hipError_t launch_rmsnorm(acache_dtype dt, const void* x, const void* g, void* y, int rows, int d,
                          float eps, hipStream_t s) {
  const bool vec = d % 8 == 0 && d <= 8192 && (uintptr_t)x % 16 == 0 && (uintptr_t)g % 16 == 0 &&
                   (uintptr_t)y % 16 == 0;
  if (dt == ACACHE_BF16 && vec)
    hipLaunchKernelGGL(rmsnorm_vec_kernel, dim3(rows), dim3(256), 0, s, (const bf16*)x, (const bf16*)g, (bf16*)y,
                       d, eps, nullptr, (int64_t)0);
  else if (dt == ACACHE_BF16)
    hipLaunchKernelGGL(rmsnorm_kernel<bf16>, dim3(rows), dim3(256), 0, s, (const bf16*)x,
                       (const bf16*)g, (bf16*)y, d, eps);
  else
    hipLaunchKernelGGL(rmsnorm_kernel<float>, dim3(rows), dim3(256), 0, s, (const float*)x,
                       (const float*)g, (float*)y, d, eps);
  return hipGetLastError();
}

bool rmsnorm_rows_ok(const void* x, const void* g, const void* y, int d) {
  return d % 8 == 0 && d <= 8192 && (uintptr_t)x % 16 == 0 && (uintptr_t)g % 16 == 0 && (uintptr_t)y % 16 == 0;
}

hipError_t launch_rmsnorm_rows(const void* x, int64_t n_src, const int32_t* src_rows, const void* g, void* y,
                               int rows, int d, float eps, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(rmsnorm_vec_kernel, dim3(rows), dim3(256), 0, s, (const bf16*)x, (const bf16*)g, (bf16*)y, d,
                     eps, src_rows, n_src);
  return hipGetLastError();
}

hipError_t launch_reduce_residual(void* x, const float* part, int splits, int M, int d,
                                  const void* g, void* y, float eps, hipStream_t s) {
  const int nc = ((d >> 3) + 255) / 256;
  auto go = [&](auto kern) {
    hipLaunchKernelGGL(kern, dim3(M), dim3(256), 0, s, (bf16*)x, part, splits, M, d, (const bf16*)g, (bf16*)y, eps);
  };
  if (nc <= 1) go(reduce_residual_kernel<1>);
  else if (nc == 2) go(reduce_residual_kernel<2>);
  else if (nc == 3) go(reduce_residual_kernel<3>);
  else go(reduce_residual_kernel<4>);
  return hipGetLastError();
}

// ---------------------------------------------------------------- rotary table
// One thread per (row, pair): the angle pos * theta_d in fp64 (theta_d =
// base^(-2d/128)), reduced and evaluated by rotary_sincos as everywhere else
// on the path; the QKV projection's epilogue reads it for all its heads.
__global__ __launch_bounds__(256) void rope_table_kernel(const int32_t* __restrict__ pos, int M, double l2b,
                                                         float* __restrict__ table) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)M * 64) return;
  const int m = (int)(i >> 6), d = (int)(i & 63);
  float sn, cs;
  rotary_sincos((double)pos[m] * exp2(-(2.0 * d / 128.0) * l2b), &sn, &cs);
  const float2 v = {cs, sn};
  reinterpret_cast<float2*>(table)[i] = v;
}

hipError_t launch_rope_table(const int32_t* pos, int M, float rope_base, float* table, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  const int64_t n = (int64_t)M * 64;
  hipLaunchKernelGGL(rope_table_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, pos, M,
                     log2((double)rope_base), table);
  return hipGetLastError();
}

hipError_t launch_q_rotary_reduce(const float* part, int splits, int n, int H, const int32_t* rows,
                                  const int32_t* pos, float rope_base, void* q, int64_t q_n_rows, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t threads = (int64_t)n * H * 16;
  hipLaunchKernelGGL(q_rotary_reduce_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s, part, splits,
                     n, H, rows, pos, rope_base, (bf16*)q, q_n_rows);
  return hipGetLastError();
}

hipError_t launch_argmax_commit(acache_dtype dt, const void* x, int64_t ld, int rows, int n, int32_t* out,
                               float* conf, const int32_t* commit_pos, int32_t* ids, int64_t ids_len, hipStream_t s) {
  const int es = dt == ACACHE_BF16 ? 2 : 4;
  const int vec = ((uintptr_t)x % 16 == 0 && (ld * es) % 16 == 0) ? 1 : 0;
  if (dt == ACACHE_BF16)
    hipLaunchKernelGGL(argmax_commit_kernel<bf16>, dim3(rows), dim3(256), 0, s, (const bf16*)x, ld, n, vec, out,
                       conf, commit_pos, ids, ids_len);
  else
    hipLaunchKernelGGL(argmax_commit_kernel<float>, dim3(rows), dim3(256), 0, s, (const float*)x, ld, n, vec, out,
                       conf, commit_pos, ids, ids_len);
  return hipGetLastError();
}

hipError_t launch_rerotate(acache_dtype dt, const void* src, int64_t src_ld, const int32_t* src_slots, void* dst,
                           int64_t dst_ld, const int32_t* dst_slots, const int32_t* delta, int n, int64_t n_slots,
                           int heads, int dh, float rope_base, hipStream_t s) {
  const double l2b = log2((double)rope_base);
  if (dt == ACACHE_BF16)
    hipLaunchKernelGGL(rerotate_kernel<bf16>, dim3(n), dim3(256), 0, s, (const bf16*)src, src_ld, src_slots,
                       (bf16*)dst, dst_ld, dst_slots, delta, n_slots, heads, dh, l2b);
  else
    hipLaunchKernelGGL(rerotate_kernel<float>, dim3(n), dim3(256), 0, s, (const float*)src, src_ld, src_slots,
                       (float*)dst, dst_ld, dst_slots, delta, n_slots, heads, dh, l2b);
  return hipGetLastError();
}

hipError_t launch_kv_deviation(acache_dtype dt, const void* kp, const void* vp, int64_t pool_ld, int64_t n_slots,
                              const int32_t* fresh, int64_t fresh_ld, const int32_t* stale, int batch, int L,
                              int width, float* scores, hipStream_t s) {
  if (dt == ACACHE_BF16)
    hipLaunchKernelGGL(kv_deviation_kernel<bf16>, dim3(L, batch), dim3(64), 0, s, (const bf16*)kp, (const bf16*)vp,
                       pool_ld, n_slots, fresh, fresh_ld, stale, L, width, scores);
  else
    hipLaunchKernelGGL(kv_deviation_kernel<float>, dim3(L, batch), dim3(64), 0, s, (const float*)kp,
                       (const float*)vp, pool_ld, n_slots, fresh, fresh_ld, stale, L, width, scores);
  return hipGetLastError();
}

hipError_t launch_threshold_commit(int batch, int block, const int32_t* pick, const float* conf, float tau,
                                  int32_t* committed, const int32_t* commit_pos, int32_t* ids, int64_t ids_len,
                                  int32_t* count, hipStream_t s) {
  hipLaunchKernelGGL(threshold_commit_kernel, dim3(batch), dim3(64), 0, s, block, pick, conf, tau, committed,
                     commit_pos, ids, ids_len, count);
  return hipGetLastError();
}

hipError_t launch_head_reduce(const float* part, int batch, int H, int L, float* scores, int init,
                              hipStream_t s) {
  const int64_t work = (int64_t)batch * L;
  hipLaunchKernelGGL(head_reduce_kernel, dim3((unsigned)((work + 31) / 32)), dim3(256), 0, s, part,
                     batch, H, L, scores, init);
  return hipGetLastError();
}

}  // namespace acache
