// Probe scoring (Section 3.2, Eq. 4-5) for the bf16 path, MFMA.
#include <algorithm>

#include "device.h"
#include "internal.h"

namespace acache {

namespace {

constexpr int kDh = 128;

typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4;

// ============================================================================
// Eq. 4-5 for one layer in one launch: the affix-only log-sum-exp of
// every masked query and the per-head column sums.
//
// A workgroup holds KG key groups of QW wavefronts; each wavefront owns 32
// masked queries (MFMA fragments of Q in registers), so a pass covers
// 32 QW queries, and key group g streams its own contiguous range of the
// affix key tiles (64 keys) through its own two LDS stages (global -> LDS
// copies, one tile ahead).  For each pass of queries:
//   sweep 1  S^T = K Q^T: online (max, sum) per query (one query per lane);
//            the key groups' statistics merge through LDS into the base-2
//            log-sum-exp (skipped under the full-softmax reading, whose
//            log-sum-exp the caller supplies);
//   sweep 2  S = Q K^T over the same keys: one key per lane, so a key's
//            mass exp2(s - lse) summed over the wavefront's queries is an
//            in-register sum and one exchange between the lane halves; the
//            QW wavefronts of a group add theirs in wavefront order through
//            LDS.
// A workgroup takes passes p = qs, qs + QS, ... of its (request, head) and
// adds them, in that order, into its own row part[b][h][qs][0..L); a fixed-
// order reduction over heads and splits then forms scores[b][j], so the
// result does not depend on timing.  Keys past the affix or with an
// out-of-range slot read zeros (their mass is exp2(-lse)).
// ============================================================================

struct ScoreFArgs {
  const bf16* q;
  int64_t q_ld;
  int64_t q_n_rows;
  const int32_t* q_rows;
  const bf16* k_pool;
  int64_t pool_ld;
  int64_t n_slots;
  const int32_t* affix_slots;
  const float* row_lse;  // full-softmax reading: [q_n_rows, H] natural log; null: affix-only (computed)
  float* part;           // [batch][H][QS][L]
  int H, Hkv, L, QS, batch;
  int cu_q[kMaxBatch + 1];
};

template <int QW, int KG>
__global__ __launch_bounds__(64 * QW * KG) void score_fused_kernel(ScoreFArgs a) {
  constexpr int kTQ = 32 * QW;                 // queries per pass
  constexpr int kTileKeys = 64;
  constexpr int kRowB = kDh * 2;               // 256 B per key row
  constexpr int kTileB = kTileKeys * kRowB;    // 16 KB
  constexpr int kDma = kTileB / 1024 / QW;     // 1 KB copies per wave and tile
  constexpr int kKeysPerWave = kTileKeys / QW;
  static_assert(kKeysPerWave == 4 * kDma, "copy split");
  __shared__ __attribute__((aligned(1024))) char ring[KG * 2 * kTileB];
  __shared__ float xch[KG > 1 ? (KG - 1) * QW * 2 * 64 : 1];  // (max, sum) of groups 1..
  __shared__ float lse_s[QW * 32];                            // base-2 LSE of the pass's queries
  __shared__ float col_x[QW > 1 ? 2 * KG * QW * 64 : 1];      // column sums per wave, two tiles

  // XCD-contiguous, head-major order of (head, request, split): the affix
  // keys of a KV head are read by every request, so they stay in one L2
  int h, b, qs;
  {
    const int nb = gridDim.x, i = blockIdx.x;
    const int q8 = nb >> 3, r8 = nb & 7, x = i & 7;
    const int t = x * q8 + min(x, r8) + (i >> 3);
    h = t / (a.batch * a.QS);
    const int rem = t - h * a.batch * a.QS;
    b = rem / a.QS;
    qs = rem - b * a.QS;
  }
  const int g = h / (a.H / a.Hkv);
  const int tid = threadIdx.x, lane = tid & 63, hl = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int gk = wave / QW, wq = wave % QW;
  const int gtid = tid - gk * 64 * QW;  // thread within the key group
  const int q0 = a.cu_q[b], nq = a.cu_q[b + 1] - q0;
  const int L = a.L;
  float* prow = a.part + (((int64_t)b * a.H + h) * a.QS + qs) * L;
  const int n_pass = (nq + kTQ - 1) / kTQ;
  if (qs >= n_pass) {
    // no queries for this split: its row adds nothing
    for (int j = tid; j < L; j += 64 * QW * KG) prow[j] = 0.f;
    return;
  }

  char* const tiles = ring + gk * 2 * kTileB;
  const int n_tiles = (L + kTileKeys - 1) / kTileKeys;
  const int t_lo = gk * n_tiles / KG, t_hi = (gk + 1) * n_tiles / KG;
  const int n_it = (n_tiles + KG - 1) / KG;  // iterations of every group (barriers line up)
  const float scale = kLog2e * rsqrtf((float)kDh);
  const int pch = lane & 15;
  const uint32_t head_b = (uint32_t)g * kRowB;
  const uint32_t ld_b = (uint32_t)a.pool_ld * 2u;

  // copies of key tile t into stage buf: this lane's keys kKeysPerWave wq +
  // 4 i + lane / 16, chunk lane % 16 at chunk position c ^ (row & 15)
  int slot_next[kDma];
  unsigned absent = 0;
  auto load_slots = [&](int t) {
#pragma unroll
    for (int i = 0; i < kDma; ++i) {
      const int j = t * kTileKeys + wq * kKeysPerWave + 4 * i + (lane >> 4);
      slot_next[i] = j < L ? a.affix_slots[j] : -1;
    }
  };
  auto issue = [&](int buf) {
    char* st = tiles + buf * kTileB;
    unsigned ab = 0;
#pragma unroll
    for (int i = 0; i < kDma; ++i) {
      const int sl = slot_next[i];
      const bool ok = sl >= 0 && sl < a.n_slots;
      ab |= (ok ? 0u : 1u) << i;
      const int r = wq * kKeysPerWave + 4 * i + (lane >> 4);
      const int ck = pch ^ (r & 15);
      dma16((const char*)a.k_pool + (ok ? (uint32_t)sl : 0u) * ld_b + head_b + ck * 16,
            st + (wq * kDma + i) * 1024);
    }
    absent = ab;
  };
  auto fix_absent = [&](int buf) {
    if (absent) {
      char* st = tiles + buf * kTileB;
      const u32x4 z = {0u, 0u, 0u, 0u};
#pragma unroll
      for (int i = 0; i < kDma; ++i)
        if ((absent >> i) & 1u) *reinterpret_cast<u32x4*>(st + (wq * kDma + i) * 1024 + lane * 16) = z;
    }
  };
  // K fragment s2 of 32-key block kb: row lane % 32, dimensions 16 s2 + 8 hl ..
  auto kfrag = [&](const char* st, int kb, int s2) {
    const int r = kb * 32 + (lane & 31);
    return *reinterpret_cast<const bf16x8*>(st + r * kRowB + (((2 * s2 + hl) ^ (r & 15)) << 4));
  };
  // runs one sweep over the group's key tiles; body(t, st) per tile
  auto sweep = [&](auto&& body) {
    if (t_lo < t_hi) {
      load_slots(t_lo);
      issue(0);
      if (t_lo + 1 < t_hi) load_slots(t_lo + 1);
    }
    for (int it = 0; it < n_it; ++it) {
      const int t = t_lo + it;
      wait_vmcnt<0>();
      fix_absent(it & 1);
      lds_barrier();
      if (t + 1 < t_hi) {
        issue((it + 1) & 1);
        if (t + 2 < t_hi) load_slots(t + 2);
      }
      body(it, t < t_hi ? t : -1, tiles + (it & 1) * kTileB);
    }
    lds_barrier();  // every group is past its last LDS read of the sweep
  };

  for (int p = qs; p < n_pass; p += a.QS) {
    // this wave's queries of pass p: Q[q][16 s + 8 hl .. +7]
    const int qi = p * kTQ + wq * 32 + (lane & 31);
    int64_t qrow = -1;
    if (qi < nq) {
      qrow = a.q_rows[q0 + qi];
      if (qrow < 0 || qrow >= a.q_n_rows) qrow = -1;
    }
    bf16x8 qf[8];
    {
      const bf16* qp = a.q + (qrow < 0 ? 0 : qrow) * a.q_ld + h * kDh + hl * 8;
#pragma unroll
      for (int s2 = 0; s2 < 8; ++s2) {
        u32x4 v = {0u, 0u, 0u, 0u};
        if (qrow >= 0) v = *reinterpret_cast<const u32x4*>(qp + s2 * 16);
        qf[s2] = __builtin_bit_cast(bf16x8, v);
      }
    }

    // ---- sweep 1: base-2 log-sum-exp of this lane's query over the affix keys
    float lse2 = INFINITY;  // absent query: exp2(s - inf) = 0
    if (a.row_lse) {
      if (qrow >= 0) lse2 = a.row_lse[qrow * a.H + h] * kLog2e;
    } else {
      float m_run = -INFINITY, l_part = 0.f;
      sweep([&](int, int t, const char* st) {
        if (t < 0) return;
        f32x16 s[2];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
          for (int r = 0; r < 16; ++r) s[kb][r] = 0.f;
#pragma unroll
          for (int s2 = 0; s2 < 8; ++s2) s[kb] = mfma32x32x16(kfrag(st, kb, s2), qf[s2], s[kb]);
        }
        // register r of block kb: key 32 kb + 8 (r / 4) + 4 hl + r % 4 of the tile
        const int kt0 = t * kTileKeys;
        float mx = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            if (kt0 + kTileKeys > L && kt0 + kb * 32 + 8 * (r >> 2) + 4 * hl + (r & 3) >= L) s[kb][r] = -INFINITY;
            mx = fmaxf(mx, s[kb][r]);
          }
        mx = fmaxf(mx, __shfl_xor(mx, 32)) * scale;
        if (mx > m_run + 8.f) {  // lazy rescale: exp2 values stay <= 2^8
          l_part *= __builtin_amdgcn_exp2f(m_run - mx);
          m_run = mx;
        }
        float ps = 0.f;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) ps += __builtin_amdgcn_exp2f(fmaf(s[kb][r], scale, -m_run));
        l_part += ps;
      });
      // merge the key groups' (max, sum) in group order, into group 0
      if constexpr (KG > 1) {
        if (gk > 0) {
          float* d = xch + ((gk - 1) * QW + wq) * 2 * 64 + lane;
          d[0] = m_run;
          d[64] = l_part;
        }
        lds_barrier();
        if (gk == 0) {
#pragma unroll
          for (int o = 1; o < KG; ++o) {
            const float* src = xch + ((o - 1) * QW + wq) * 2 * 64 + lane;
            const float m_o = src[0];
            const float m_new = fmaxf(m_run, m_o);
            const float a_self = m_run == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_run - m_new);
            const float a_o = m_o == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_o - m_new);
            l_part = l_part * a_self + src[64] * a_o;
            m_run = m_new;
          }
        }
      }
      const float l_tot = l_part + __shfl_xor(l_part, 32);
      if (qrow >= 0) lse2 = m_run + __log2f(l_tot);
    }
    // the pass's LSEs to every wave: query row 8 (r / 4) + 4 hl + r % 4 of
    // sweep 2's accumulator
    if (gk == 0 && hl == 0) lse_s[wq * 32 + (lane & 31)] = lse2;
    lds_barrier();
    float lq[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) lq[r] = lse_s[wq * 32 + 8 * (r >> 2) + 4 * hl + (r & 3)];

    // ---- sweep 2: column sums over this pass's queries
    const bool first = p == qs;
    auto flush = [&](int it_prev, int t_prev) {
      // group gk's tile t_prev: the QW waves' sums, in wave order, by wave 0
      if constexpr (QW > 1) {
        if (wq == 0 && t_prev >= 0) {
          const float* cx = col_x + ((it_prev & 1) * KG + gk) * QW * 64 + lane;
          float tot = 0.f;
#pragma unroll
          for (int w = 0; w < QW; ++w) tot += cx[w * 64];
          const int j = t_prev * kTileKeys + lane;
          if (j < L) prow[j] = first ? tot : prow[j] + tot;
        }
      }
    };
    int prev_it = -1, prev_t = -1;
    sweep([&](int it, int t, const char* st) {
      flush(prev_it, prev_t);  // the previous tile's wave sums are in LDS (barrier passed)
      prev_it = it;
      prev_t = t;
      if (t < 0) return;
      float cs[2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        f32x16 s = {};
#pragma unroll
        for (int s2 = 0; s2 < 8; ++s2) s = mfma32x32x16(qf[s2], kfrag(st, kb, s2), s);
        float c = 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) c += __builtin_amdgcn_exp2f(fmaf(s[r], scale, -lq[r]));
        cs[kb] = c + __shfl_xor(c, 32);
      }
      // lane l: key 32 (l / 32) + l % 32 of the tile
      const float mine = hl ? cs[1] : cs[0];
      if constexpr (QW > 1) {
        col_x[((it & 1) * KG + gk) * QW * 64 + wq * 64 + lane] = mine;
      } else {
        const int j = t * kTileKeys + lane;
        if (j < L) prow[j] = first ? mine : prow[j] + mine;
      }
    });
    flush(prev_it, prev_t);  // sweep() ended with a barrier
    lds_barrier();           // lse_s and col_x are rewritten by the next pass
  }
}

}  // namespace

hipError_t launch_score_fused_bf16(int batch, const int* cu_q, int H, int Hkv, const void* q, int64_t q_ld,
                                   int64_t q_n_rows, const int32_t* q_rows, const void* k_pool, int64_t pool_ld,
                                   int64_t n_slots, const int32_t* affix_slots, int L, const float* row_lse,
                                   float* part, size_t part_bytes, int* rows_per_request, hipStream_t s) {
  ScoreFArgs a = {};
  a.q = (const bf16*)q;
  a.q_ld = q_ld;
  a.q_n_rows = q_n_rows;
  a.q_rows = q_rows;
  a.k_pool = (const bf16*)k_pool;
  a.pool_ld = pool_ld;
  a.n_slots = n_slots;
  a.affix_slots = affix_slots;
  a.row_lse = row_lse;
  a.part = part;
  a.H = H;
  a.Hkv = Hkv;
  a.L = L;
  a.batch = batch;
  int max_q = 0;
  for (int b = 0; b <= batch; ++b) a.cu_q[b] = cu_q[b];
  for (int b = 0; b < batch; ++b) max_q = std::max(max_q, cu_q[b + 1] - cu_q[b]);
  const size_t row_bytes = (size_t)batch * H * L * sizeof(float);
  if (row_bytes == 0 || row_bytes > part_bytes) return hipErrorInvalidValue;
  // grids of a workgroup per CU or more: 128 queries per pass (2 key groups
  // of 4 waves), one split (at 256 request-heads 2% faster per C3 step than
  // 32 queries per pass); small ones: 32 queries per pass (4 key groups of
  // one wave) and as many splits of the passes as fill the chip and the region
  const bool big = (int64_t)batch * H >= 256;
  const int tq = big ? 128 : 32;
  const int passes = std::max(1, (max_q + tq - 1) / tq);
  int qs = 1;
  if (!big)
    while (qs * 2 <= passes && (size_t)(qs * 2) * row_bytes <= part_bytes && (int64_t)batch * H * qs < 256) qs *= 2;
  a.QS = qs;
  *rows_per_request = H * qs;
  const int grid = batch * H * qs;
  if (big)
    hipLaunchKernelGGL((score_fused_kernel<4, 2>), dim3(grid), dim3(512), 0, s, a);
  else
    hipLaunchKernelGGL((score_fused_kernel<1, 4>), dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace acache
