// Probe scoring, column-sum pass (Section 3.2, Eq. 4-5), bf16 MFMA.
//
// One workgroup per (request, 64 affix keys, head), kQSplit wavefronts that
// take the request's masked queries in interleaved tiles of 32 and add their
// column sums in a fixed order at the end.  Each wavefront keeps the keys' K
// fragments in registers and streams its query tiles: S = Q K^T with Q as the MFMA A operand puts one key column per lane
// (the 16 accumulator registers are 16 queries), so a key's attention mass
// over the tile is an in-register sum; the two lane halves are combined once
// at the end.  a = exp2(s * log2(e) / sqrt(d_h) - lse2) with the row's
// log-sum-exp over the affix keys (the Eq. 4 normalisation) or over all keys.
// The per-head column sums go to a workspace; a separate pass adds them over
// heads in a fixed order, so scores are bit-reproducible.
#include "device.h"
#include "internal.h"

namespace acache {

namespace {

constexpr int kDh = 128;
constexpr int kQSplit = 4;  // wavefronts per workgroup, each a quarter of the query tiles
constexpr int kLseStage = 2048;  // queries per request whose LSE is staged in LDS

typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4;

struct ColsumArgs {
  const bf16* q;
  int64_t q_ld;
  int64_t q_n_rows;
  const int32_t* q_rows;
  const bf16* k_pool;
  int64_t pool_ld;
  int64_t n_slots;
  const int32_t* affix_slots;
  const float* lse;
  int lse_by_qrow;
  float* part;  // [batch][H][L]
  int H, Hkv, L;
  int cu_q[kMaxBatch + 1];
};

__global__ __launch_bounds__(64 * kQSplit) void colsum_kernel(ColsumArgs a) {
  const int kt = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, hl = lane >> 5;
  constexpr int STEP = 32 * kQSplit;  // query stride between a wavefront's tiles
  __shared__ float red[kQSplit][64];
  __shared__ float lse_s[kLseStage];
  const int g = h / (a.H / a.Hkv);
  const float scale = kLog2e * rsqrtf((float)kDh);

  // B operand: K[key = kt*64 + 32 sub + lane%32][16 s + 8 hl .. +7]
  bf16x8 kf[2][8];
#pragma unroll
  for (int sub = 0; sub < 2; ++sub) {
    const int j = kt * 64 + sub * 32 + (lane & 31);
    int64_t slot = -1;
    if (j < a.L) {
      slot = a.affix_slots[j];
      if (slot < 0 || slot >= a.n_slots) slot = -1;
    }
    const bf16* kp = a.k_pool + (slot < 0 ? 0 : slot) * a.pool_ld + (int64_t)g * kDh + hl * 8;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (slot >= 0) v = *reinterpret_cast<const u32x4*>(kp + s * 16);
      kf[sub][s] = __builtin_bit_cast(bf16x8, v);
    }
  }

  const int q0 = a.cu_q[b], nq = a.cu_q[b + 1] - q0;
  float col[2] = {0.f, 0.f};
  // query tile t: A operand Q[query t + lane%32][16 s + 8 hl .. +7].  Row
  // indices run two tiles ahead and Q fragments one tile ahead of the MFMAs.
  auto row_of = [&](int t) -> int64_t {
    const int qi = t + (lane & 31);
    if (qi >= nq) return -1;
    const int64_t r = a.q_rows[q0 + qi];
    return (r >= 0 && r < a.q_n_rows) ? r : -1;
  };
  auto load_q = [&](int64_t row, bf16x8* qf) {
    const bf16* qp = a.q + (row < 0 ? 0 : row) * a.q_ld + (int64_t)h * kDh + hl * 8;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (row >= 0) v = *reinterpret_cast<const u32x4*>(qp + s * 16);
      qf[s] = __builtin_bit_cast(bf16x8, v);
    }
  };
  bf16x8 qcur[8], qnext[8];
  const int t0 = wave * 32;
  int64_t row_next = row_of(t0 + STEP);
  load_q(row_of(t0), qcur);
  // the LSE (base 2) of every query of the request, staged in LDS with the
  // first loads in flight (+inf for absent rows: exp2(-inf) = 0)
  const bool staged = nq <= kLseStage;
  if (staged) {
    for (int i = threadIdx.x; i < nq; i += 64 * kQSplit) {
      const int64_t idx = a.lse_by_qrow ? (int64_t)(q0 + i) : (int64_t)a.q_rows[q0 + i];
      const bool ok = a.lse_by_qrow || (idx >= 0 && idx < a.q_n_rows);
      lse_s[i] = ok ? a.lse[idx * a.H + h] * kLog2e : INFINITY;
    }
    __syncthreads();
  }
  for (int t = t0; t < nq; t += STEP) {
    if (t + STEP < nq) load_q(row_next, qnext);
    if (t + 2 * STEP < nq) row_next = row_of(t + 2 * STEP);
    // log-sum-exp (base 2) of the 16 queries this lane's registers hold.
    // The loads are unconditional (clamped indices) so that all 16 are in
    // flight together; absent queries then take +inf, i.e. exp2(-inf) = 0.
    float lse2[16];
    if (staged) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int qq = t + 8 * (r >> 2) + 4 * hl + (r & 3);
        lse2[r] = qq < nq ? lse_s[qq] : INFINITY;
      }
    } else {
      int64_t lidx[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int qq = t + 8 * (r >> 2) + 4 * hl + (r & 3);
        const int qc = min(qq, nq - 1);
        lidx[r] = a.lse_by_qrow ? (int64_t)(q0 + qc) : (int64_t)a.q_rows[q0 + qc];
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int qq = t + 8 * (r >> 2) + 4 * hl + (r & 3);
        const bool ok = qq < nq && (a.lse_by_qrow || (lidx[r] >= 0 && lidx[r] < a.q_n_rows));
        const float v = a.lse[(ok ? lidx[r] : 0) * a.H + h];
        lse2[r] = ok ? v * kLog2e : INFINITY;
      }
    }
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
      f32x16 acc;
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[r] = 0.f;
#pragma unroll
      for (int s = 0; s < 8; ++s) acc = mfma32x32x16(qcur[s], kf[sub][s], acc);
      float cs = 0.f;
#pragma unroll
      for (int r = 0; r < 16; ++r) cs += exp2f(acc[r] * scale - lse2[r]);
      col[sub] += cs;
    }
#pragma unroll
    for (int s = 0; s < 8; ++s) qcur[s] = qnext[s];
  }
  // key (lane & 31) + 32 sub: lane halves, then the wavefronts in order
#pragma unroll
  for (int sub = 0; sub < 2; ++sub) {
    const float tot = col[sub] + __shfl_xor(col[sub], 32);
    if (hl == sub) red[wave][lane] = tot;
  }
  __syncthreads();
  if (wave == 0) {
    float tot = red[0][lane];
#pragma unroll
    for (int w = 1; w < kQSplit; ++w) tot += red[w][lane];
    const int j = kt * 64 + lane;
    if (j < a.L) a.part[((int64_t)b * a.H + h) * a.L + j] = tot;
  }
}

}  // namespace

hipError_t launch_score_colsum_bf16(int batch, const int* cu_q, int H, int Hkv, const void* q,
                                    int64_t q_ld, int64_t q_n_rows, const int32_t* q_rows,
                                    const void* k_pool, int64_t pool_ld, int64_t n_slots,
                                    const int32_t* affix_slots, int L, const float* lse,
                                    int lse_by_qrow, float* part, hipStream_t s) {
  ColsumArgs a = {};
  a.q = (const bf16*)q;
  a.q_ld = q_ld;
  a.q_n_rows = q_n_rows;
  a.q_rows = q_rows;
  a.k_pool = (const bf16*)k_pool;
  a.pool_ld = pool_ld;
  a.n_slots = n_slots;
  a.affix_slots = affix_slots;
  a.lse = lse;
  a.lse_by_qrow = lse_by_qrow;
  a.part = part;
  a.H = H;
  a.Hkv = Hkv;
  a.L = L;
  for (int b = 0; b <= batch; ++b) a.cu_q[b] = cu_q[b];
  hipLaunchKernelGGL(colsum_kernel, dim3((L + 63) / 64, H, batch), dim3(64 * kQSplit), 0, s, a);
  return hipGetLastError();
}

}  // namespace acache
