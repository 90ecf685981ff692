// fp32 path of the recompute block.  On gfx950 the fp32 matrix and fp32
// vector peaks are equal (157 TFLOP/s), so the fp32 contractions use LDS-tiled
// vector FMA instead of the 32x32x2 fp32 MFMA.  Rotary angles are reduced in
// fp64 so the fp32 outputs stay within a few ulp at any position.
#include "device.h"
#include "internal.h"

namespace acache {

namespace {

// ---------------------------------------------------------------- GEMM  C = X W^T (+ C)
constexpr int TM = 64, TN = 64, TK = 16;

__global__ __launch_bounds__(256) void gemm_f32_kernel(const float* __restrict__ X, const float* __restrict__ W,
                                                       float* __restrict__ C, int64_t ldc, int M, int N,
                                                       int K, int accumulate) {
  __shared__ float sA[TK][TM + 4];
  __shared__ float sB[TK][TN + 4];
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int m0 = blockIdx.y * TM, n0 = blockIdx.x * TN;
  float c[4][4] = {};
  // the next K tile is loaded into registers while the current one computes
  float ra[4], rb[4];
  auto load = [&](int k0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int idx = threadIdx.x + i * 256;
      const int r = idx / TK, kk = idx % TK;
      const int m = m0 + r, n = n0 + r, k = k0 + kk;
      ra[i] = (m < M && k < K) ? X[(int64_t)m * K + k] : 0.f;
      rb[i] = (n < N && k < K) ? W[(int64_t)n * K + k] : 0.f;
    }
  };
  load(0);
  for (int k0 = 0; k0 < K; k0 += TK) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int idx = threadIdx.x + i * 256;
      const int r = idx / TK, kk = idx % TK;
      sA[kk][r] = ra[i];
      sB[kk][r] = rb[i];
    }
    __syncthreads();
    if (k0 + TK < K) load(k0 + TK);
#pragma unroll
    for (int kk = 0; kk < TK; ++kk) {
      float av[4], bv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) av[i] = sA[kk][ty + 16 * i];
#pragma unroll
      for (int j = 0; j < 4; ++j) bv[j] = sB[kk][tx + 16 * j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) c[i][j] = fmaf(av[i], bv[j], c[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int m = m0 + ty + 16 * i, n = n0 + tx + 16 * j;
      if (m < M && n < N) {
        float* p = C + (int64_t)m * ldc + n;
        *p = accumulate ? *p + c[i][j] : c[i][j];
      }
    }
}

// ---------------------------------------------------------------- rotary + K/V store
__global__ __launch_bounds__(256) void rope_scatter_f32_kernel(const float* __restrict__ qkv, int H, int Hkv,
                                                               int dh, const int32_t* __restrict__ pos,
                                                               float rope_base, float* __restrict__ q_out,
                                                               const int32_t* __restrict__ wslots,
                                                               float* __restrict__ kp, float* __restrict__ vp,
                                                               int64_t pool_ld, int64_t n_slots) {
  const int64_t m = blockIdx.x;
  const int half = dh / 2;
  const int width = (H + 2 * Hkv) * dh;
  const float* row = qkv + m * width;
  const int64_t slot = wslots[m];
  const bool slot_ok = slot >= 0 && slot < n_slots;
  const double p = (double)pos[m];
  // rotated pairs of the Q and K heads
  for (int c = threadIdx.x; c < (H + Hkv) * half; c += blockDim.x) {
    const int head = c / half, i = c % half;
    const double ang = p * exp2(-(2.0 * i / dh) * log2((double)rope_base));
    double sn, cs;
    sincos(ang, &sn, &cs);
    const float x1 = row[head * dh + i], x2 = row[head * dh + i + half];
    const float o1 = (float)(x1 * cs - x2 * sn), o2 = (float)(x2 * cs + x1 * sn);
    if (head < H) {
      q_out[m * H * dh + head * dh + i] = o1;
      q_out[m * H * dh + head * dh + i + half] = o2;
    } else if (slot_ok) {
      const int kh = head - H;
      kp[slot * pool_ld + kh * dh + i] = o1;
      kp[slot * pool_ld + kh * dh + i + half] = o2;
    }
  }
  if (slot_ok)
    for (int c = threadIdx.x; c < Hkv * dh; c += blockDim.x) vp[slot * pool_ld + c] = row[(H + Hkv) * dh + c];
}

__global__ __launch_bounds__(256) void swiglu_f32_kernel(const float* __restrict__ gu, int M, int F,
                                                         float* __restrict__ h) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= (int64_t)M * F) return;
  const int64_t m = t / F, f = t % F;
  const float g = gu[m * 2 * F + f], u = gu[m * 2 * F + F + f];
  h[t] = g / (1.f + expf(-g)) * u;
}

// ---------------------------------------------------------------- attention (one wave per row and head)
__device__ __forceinline__ float dot_row(const float* __restrict__ sq, const float* __restrict__ k, int dh) {
  float s = 0.f;
  for (int d = 0; d < dh; ++d) s = fmaf(sq[d], k[d], s);
  return s;
}

struct RowsArgs {
  int batch;
  int row_start[kMaxBatch + 1];
  int key_start[kMaxBatch + 1];
  int key_len[kMaxBatch + 1];
};

__device__ __forceinline__ int request_of(const RowsArgs& a, int row) {
  int lo = 0, hi = a.batch - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.row_start[mid] <= row) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Log-sum-exp (natural) of row `qrow`, head h over the keys named by slots.
__device__ float row_lse(const float* sq, const int32_t* slots, int S, const float* kp, int64_t pool_ld,
                         int64_t n_slots, int64_t koff, int dh, float scale) {
  const int lane = threadIdx.x;
  float m = -INFINITY, l = 0.f;
  for (int j = lane; j < S; j += 64) {
    const int64_t sl = slots[j];
    const float z = (sl >= 0 && sl < n_slots) ? dot_row(sq, kp + sl * pool_ld + koff, dh) * scale : 0.f;
    const float mn = fmaxf(m, z);
    l = l * expf(m - mn) + expf(z - mn);
    m = mn;
  }
  const float M = wave_max(m);
  l = (m == -INFINITY) ? 0.f : l * expf(m - M);
  return M + logf(wave_sum(l));
}

__global__ __launch_bounds__(64) void attention_f32_kernel(RowsArgs a, int H, int Hkv, int dh,
                                                           const float* __restrict__ q,
                                                           const int32_t* __restrict__ read_slots,
                                                           const float* __restrict__ kp,
                                                           const float* __restrict__ vp, int64_t pool_ld,
                                                           int64_t n_slots, float* __restrict__ out,
                                                           float* __restrict__ lse) {
  __shared__ float sq[128];
  __shared__ float sp[64];
  const int row = blockIdx.x, h = blockIdx.y, lane = threadIdx.x;
  const int b = request_of(a, row);
  const int g = h / (H / Hkv);
  const int S = a.key_len[b];
  const int32_t* slots = read_slots + a.key_start[b];
  const int64_t koff = (int64_t)g * dh;
  for (int d = lane; d < dh; d += 64) sq[d] = q[(int64_t)row * H * dh + h * dh + d];
  __syncthreads();
  const float scale = rsqrtf((float)dh);
  const float L = row_lse(sq, slots, S, kp, pool_ld, n_slots, koff, dh, scale);
  float o0 = 0.f, o1 = 0.f;
  for (int c = 0; c < S; c += 64) {
    const int j = c + lane;
    float pj = 0.f;
    if (j < S) {
      const int64_t sl = slots[j];
      const float z = (sl >= 0 && sl < n_slots) ? dot_row(sq, kp + sl * pool_ld + koff, dh) * scale : 0.f;
      pj = expf(z - L);
    }
    sp[lane] = pj;
    __syncthreads();
    const int n = min(64, S - c);
    for (int jj = 0; jj < n; ++jj) {
      const int64_t sl = slots[c + jj];
      if (sl < 0 || sl >= n_slots) continue;
      const float* vr = vp + sl * pool_ld + koff;
      if (lane < dh) o0 = fmaf(sp[jj], vr[lane], o0);
      if (lane + 64 < dh) o1 = fmaf(sp[jj], vr[lane + 64], o1);
    }
    __syncthreads();
  }
  float* op = out + (int64_t)row * H * dh + h * dh;
  if (lane < dh) op[lane] = o0;
  if (lane + 64 < dh) op[lane + 64] = o1;
  if (lse && lane == 0) lse[(int64_t)row * H + h] = L;
}

// ---------------------------------------------------------------- probe scores (Eq. 4-5)
__global__ __launch_bounds__(64) void score_lse_f32_kernel(int H, int Hkv, int dh, const float* __restrict__ q,
                                                           int64_t q_ld, int64_t q_n_rows,
                                                           const int32_t* __restrict__ q_rows,
                                                           const float* __restrict__ kp, int64_t pool_ld,
                                                           int64_t n_slots, const int32_t* __restrict__ affix_slots,
                                                           int L, float* __restrict__ lse_out) {
  __shared__ float sq[128];
  const int i = blockIdx.x, h = blockIdx.y, lane = threadIdx.x;
  const int g = h / (H / Hkv);
  int64_t row = q_rows[i];
  const bool ok = row >= 0 && row < q_n_rows;
  for (int d = lane; d < dh; d += 64) sq[d] = ok ? q[row * q_ld + h * dh + d] : 0.f;
  __syncthreads();
  const float v = row_lse(sq, affix_slots, L, kp, pool_ld, n_slots, (int64_t)g * dh, dh, rsqrtf((float)dh));
  if (lane == 0) lse_out[(int64_t)i * H + h] = v;
}

__global__ __launch_bounds__(64) void score_colsum_f32_kernel(RowsArgs a, int H, int Hkv, int dh,
                                                              const float* __restrict__ q, int64_t q_ld,
                                                              int64_t q_n_rows, const int32_t* __restrict__ q_rows,
                                                              const float* __restrict__ kp, int64_t pool_ld,
                                                              int64_t n_slots, const int32_t* __restrict__ affix_slots,
                                                              int L, const float* __restrict__ lse, int lse_by_qrow,
                                                              float* __restrict__ part) {
  __shared__ float sq[128];
  const int kt = blockIdx.x, h = blockIdx.y, b = blockIdx.z, lane = threadIdx.x;
  const int g = h / (H / Hkv);
  const int j = kt * 64 + lane;
  int64_t sl = -1;
  if (j < L) {
    sl = affix_slots[j];
    if (sl < 0 || sl >= n_slots) sl = -1;
  }
  const float* krow = kp + (sl < 0 ? 0 : sl) * pool_ld + (int64_t)g * dh;
  const float scale = rsqrtf((float)dh);
  float acc = 0.f;
  for (int qi = a.row_start[b]; qi < a.row_start[b + 1]; ++qi) {
    const int64_t row = q_rows[qi];
    const bool ok = row >= 0 && row < q_n_rows;
    __syncthreads();
    for (int d = lane; d < dh; d += 64) sq[d] = ok ? q[row * q_ld + h * dh + d] : 0.f;
    __syncthreads();
    if (!ok || sl < 0) continue;
    const float z = dot_row(sq, krow, dh) * scale;
    const float l = lse[(lse_by_qrow ? (int64_t)qi : row) * H + h];
    acc += expf(z - l);
  }
  if (j < L) part[((int64_t)b * H + h) * L + j] = acc;
}

RowsArgs rows_args(const int* starts, int batch) {
  RowsArgs a = {};
  a.batch = batch;
  for (int b = 0; b <= batch; ++b) a.row_start[b] = starts[b];
  return a;
}

}  // namespace

hipError_t launch_gemm_f32(const float* X, const float* W, float* C, int64_t ldc, int M, int N,
                           int K, int accumulate, hipStream_t s) {
  hipLaunchKernelGGL(gemm_f32_kernel, dim3((N + TN - 1) / TN, (M + TM - 1) / TM), dim3(256), 0, s, X,
                     W, C, ldc, M, N, K, accumulate);
  return hipGetLastError();
}

hipError_t launch_rope_scatter_f32(const float* qkv, int M, int H, int Hkv, int dh,
                                   const int32_t* pos, float rope_base, float* q_out,
                                   const int32_t* write_slots, float* k_pool, float* v_pool,
                                   int64_t pool_ld, int64_t n_slots, hipStream_t s) {
  hipLaunchKernelGGL(rope_scatter_f32_kernel, dim3(M), dim3(256), 0, s, qkv, H, Hkv, dh, pos, rope_base,
                     q_out, write_slots, k_pool, v_pool, pool_ld, n_slots);
  return hipGetLastError();
}

hipError_t launch_swiglu_f32(const float* gu, int M, int F, float* h, hipStream_t s) {
  const int64_t n = (int64_t)M * F;
  hipLaunchKernelGGL(swiglu_f32_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, gu, M, F, h);
  return hipGetLastError();
}

hipError_t launch_attention_f32(const Ragged& rg, int H, int Hkv, int dh, const float* q,
                                const int32_t* read_slots, const float* k_pool,
                                const float* v_pool, int64_t pool_ld, int64_t n_slots, float* out,
                                float* lse, hipStream_t s) {
  RowsArgs a = rows_args(rg.cu_rows, rg.batch);
  for (int b = 0; b < rg.batch; ++b) {
    a.key_start[b] = rg.cu_keys[b];
    a.key_len[b] = rg.cu_keys[b + 1] - rg.cu_keys[b];
  }
  const int rows = rg.cu_rows[rg.batch];
  if (rows == 0) return hipSuccess;
  hipLaunchKernelGGL(attention_f32_kernel, dim3(rows, H), dim3(64), 0, s, a, H, Hkv, dh, q, read_slots,
                     k_pool, v_pool, pool_ld, n_slots, out, lse);
  return hipGetLastError();
}

hipError_t launch_score_lse_f32(int batch, const int* cu_q, int H, int Hkv, int dh, const float* q,
                                int64_t q_ld, int64_t q_n_rows, const int32_t* q_rows,
                                const float* k_pool, int64_t pool_ld, int64_t n_slots,
                                const int32_t* affix_slots, int L, float* lse_out, hipStream_t s) {
  const int n = cu_q[batch];
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(score_lse_f32_kernel, dim3(n, H), dim3(64), 0, s, H, Hkv, dh, q, q_ld, q_n_rows,
                     q_rows, k_pool, pool_ld, n_slots, affix_slots, L, lse_out);
  return hipGetLastError();
}

hipError_t launch_score_colsum_f32(int batch, const int* cu_q, int H, int Hkv, int dh,
                                   const float* q, int64_t q_ld, int64_t q_n_rows,
                                   const int32_t* q_rows, const float* k_pool, int64_t pool_ld,
                                   int64_t n_slots, const int32_t* affix_slots, int L,
                                   const float* lse, int lse_by_qrow, float* part, hipStream_t s) {
  RowsArgs a = rows_args(cu_q, batch);
  hipLaunchKernelGGL(score_colsum_f32_kernel, dim3((L + 63) / 64, H, batch), dim3(64), 0, s, a, H, Hkv, dh,
                     q, q_ld, q_n_rows, q_rows, k_pool, pool_ld, n_slots, affix_slots, L, lse, lse_by_qrow,
                     part);
  return hipGetLastError();
}

}  // namespace acache
