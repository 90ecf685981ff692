// Probe scoring, column-sum pass (Section 3.2, Eq. 4-5), bf16 MFMA.
//
// One workgroup per (request, head, 64 W affix keys): each wavefront keeps the
// K fragments of its 64 keys in registers and sweeps all of the request's
// masked queries, whose Q rows and LSEs are staged in LDS once per workgroup.
// S = Q K^T with Q as the MFMA A operand puts one key column per lane (the
// 16 accumulator registers are 16 queries), so a key's attention mass over a
// query tile is an in-register sum; the two lane halves are combined once at
// the end.  a = exp2(s * log2(e) / sqrt(d_h) - lse2) with the row's
// log-sum-exp over the affix keys (the Eq. 4 normalisation) or over all keys.
// The per-head column sums go to a workspace; a separate pass adds them over
// heads in a fixed order, so scores are bit-reproducible.
#include "device.h"
#include "internal.h"

namespace acache {

namespace {

constexpr int kDh = 128;

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

// One workgroup per (request, head, 256 affix keys): wavefront w owns keys
// 64 w .. 64 w + 63 (its K fragments in registers) and every wavefront
// sweeps all of the request's masked queries.  The queries' Q rows and base-2
// LSEs are staged in LDS, kQChunk queries at a time, so each is read from
// memory once per 256 keys.  S = Q K^T with Q as the A operand puts one key
// per lane: a key's sum over queries is an in-register sum over the
// accumulator rows, then one exchange between the lane halves, in a fixed
// order (query tiles ascending).
constexpr int kQChunk = 256;                   // queries staged per pass
constexpr int kQRowB = kDh * 2;                // 256 B per staged query row

// W wavefronts (64 W keys) per workgroup.
template <int W>
__global__ __launch_bounds__(64 * W, 2) void colsum_kernel(ColsumArgs a) {
  constexpr int kKeysPerWg = 64 * W;
  const int kb0 = blockIdx.x * kKeysPerWg, h = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, hl = lane >> 5;
  __shared__ __attribute__((aligned(16))) char q_s[kQChunk * kQRowB];
  __shared__ float lse_s[kQChunk];
  const int g = h / (a.H / a.Hkv);
  const float scale = kLog2e * rsqrtf((float)kDh);

  // B operand: K[key = kb0 + 64 wave + 32 sub + lane%32][16 s + 8 hl .. +7]
  bf16x8 kf[2][8];
#pragma unroll
  for (int sub = 0; sub < 2; ++sub) {
    const int j = kb0 + wave * 64 + sub * 32 + (lane & 31);
    int64_t slot = -1;
    if (j < a.L) {
      slot = a.affix_slots[j];
      if (slot < 0 || slot >= a.n_slots) slot = -1;
    }
    const bf16* kp = a.k_pool + (slot < 0 ? 0 : slot) * a.pool_ld + (int64_t)g * kDh + hl * 8;
#pragma unroll
    for (int s2 = 0; s2 < 8; ++s2) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (slot >= 0) v = *reinterpret_cast<const u32x4*>(kp + s2 * 16);
      kf[sub][s2] = __builtin_bit_cast(bf16x8, v);
    }
  }

  const int q0 = a.cu_q[b], nq = a.cu_q[b + 1] - q0;
  float col[2] = {0.f, 0.f};
  // staged row r: 16-byte chunk c at c ^ (r & 15), so the 16 rows one
  // quarter-wave reads land in 16 distinct chunk positions
  const int fr = lane & 31;  // this lane's row within a 32-query tile
  for (int c0 = 0; c0 < nq; c0 += kQChunk) {
    const int nc = min(kQChunk, nq - c0);
    if (c0 > 0) __syncthreads();  // the previous chunk is no longer read
    // Q rows: 16 threads per row, one 16-byte chunk each; the loads of a
    // batch of 16 rows per thread are issued before its first store (clamped
    // rows, absent ones stored as 0)
    constexpr int kRowsPerPass = 64 * W / 16;
    constexpr int kPasses = kQChunk / kRowsPerPass;
    constexpr int kBatch = kPasses < 16 ? kPasses : 16;
#pragma unroll
    for (int it0 = 0; it0 < kPasses; it0 += kBatch) {
      u32x4 qv[kBatch];
      bool qok[kBatch];
#pragma unroll
      for (int i = 0; i < kBatch; ++i) {
        const int r = (it0 + i) * kRowsPerPass + (tid >> 4);
        const int64_t row = a.q_rows[q0 + c0 + min(r, nc - 1)];
        qok[i] = r < nc && row >= 0 && row < a.q_n_rows;
        const int64_t rowc = qok[i] ? row : 0;
        qv[i] = *reinterpret_cast<const u32x4*>(a.q + rowc * a.q_ld + (int64_t)h * kDh + (tid & 15) * 8);
      }
#pragma unroll
      for (int i = 0; i < kBatch; ++i) {
        const int r = (it0 + i) * kRowsPerPass + (tid >> 4);
        const u32x4 z = {0u, 0u, 0u, 0u};
        *reinterpret_cast<u32x4*>(q_s + r * kQRowB + (((tid & 15) ^ (r & 15)) << 4)) = qok[i] ? qv[i] : z;
      }
    }
    // base-2 LSE of each query (+inf for absent rows: exp2(-inf) = 0)
    for (int i = tid; i < kQChunk; i += 64 * W) {
      float v = INFINITY;
      if (i < nc) {
        const int64_t idx = a.lse_by_qrow ? (int64_t)(q0 + c0 + i) : (int64_t)a.q_rows[q0 + c0 + i];
        if (a.lse_by_qrow || (idx >= 0 && idx < a.q_n_rows)) v = a.lse[idx * a.H + h] * kLog2e;
      }
      lse_s[i] = v;
    }
    __syncthreads();
    for (int t = 0; t < nc; t += 32) {
      // A operand: Q[query t + lane%32][16 s + 8 hl .. +7]
      bf16x8 qf[8];
      const char* qrow = q_s + (t + fr) * kQRowB;
#pragma unroll
      for (int s2 = 0; s2 < 8; ++s2)
        qf[s2] = *reinterpret_cast<const bf16x8*>(qrow + (((2 * s2 + hl) ^ fr) & 15) * 16);
      float lse2[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) lse2[r] = lse_s[t + 8 * (r >> 2) + 4 * hl + (r & 3)];
      f32x16 acc0, acc1;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        acc0[r] = 0.f;
        acc1[r] = 0.f;
      }
#pragma unroll
      for (int s2 = 0; s2 < 8; ++s2) {
        acc0 = mfma32x32x16(qf[s2], kf[0][s2], acc0);
        acc1 = mfma32x32x16(qf[s2], kf[1][s2], acc1);
      }
      float cs0 = 0.f, cs1 = 0.f;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        cs0 += exp2f(acc0[r] * scale - lse2[r]);
        cs1 += exp2f(acc1[r] * scale - lse2[r]);
      }
      col[0] += cs0;
      col[1] += cs1;
    }
  }
  // key 32 sub + lane%32 of this wave: the two lane halves, then one store
#pragma unroll
  for (int sub = 0; sub < 2; ++sub) {
    const float tot = col[sub] + __shfl_xor(col[sub], 32);
    const int j = kb0 + wave * 64 + sub * 32 + (lane & 31);
    if (hl == sub && j < a.L) a.part[((int64_t)b * a.H + h) * a.L + j] = tot;
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
  // 4 wavefronts (256 keys) per workgroup; 2-wavefront workgroups were
  // slower even where they double the workgroup count (one request)
  hipLaunchKernelGGL(colsum_kernel<4>, dim3((L + 255) / 256, H, batch), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace acache
