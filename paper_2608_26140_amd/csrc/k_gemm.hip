// bf16 MFMA GEMM for the recompute rows: C[m, n] = sum_k X[m, k] W[n, k].
//
// Both operands are K-contiguous (activations [M, K], weights [N, K]), so
// each lane loads 16-byte runs along K straight into the MFMA operand
// layout.  The weight tile feeds the MFMA A operand and the activation tile
// the B operand: the accumulator then holds, per lane, one activation row
// and runs of 4 consecutive output columns, which gives 8-byte output stores
// and puts both halves of every rotary pair (columns d and d + 64 of one
// head) in the same lane.
//
// Workgroup tiles: 256 weight rows x 256 activation rows, 4 waves (one per
// SIMD) of 128 x 128 on MFMA 16x16x32 with the accumulators in AGPRs, the
// weight rows of three 64-wide K steps and the activation rows of two in
// LDS (gemm_bf16_w4_kernel); or, where it
// leaves fewer CUs idle, 256 x 128 with 8 waves (two per SIMD) of 128 x 32
// on MFMA 32x32x16 and a ping-pong schedule over 32-wide K units
// (gemm_bf16_kernel).  Both are fed by buffer -> LDS copies (no staging
// registers).  The rotary epilogue reads each row's (cos, sin) table,
// computed once per projection by launch_rope_table.  Workgroups are
// renumbered so that each XCD (8 per chip, own L2) receives a contiguous
// run of tiles with the M index fastest: the tiles sharing one weight tile
// run on the same L2.
//
// Schedules.  Data-parallel: one tile (or one K split of a tile) per
// workgroup.  Stream-K, for the recompute's small row counts where the
// tile count is not a multiple of the CU count: the full rounds of tiles run
// data-parallel, and the K steps of the remaining tiles are dealt evenly to
// all workgroups.  A workgroup whose K range covers only part of a tile
// writes its fp32 accumulators to a workspace slot; a fixup kernel (one
// wave per wave-tile) sums the pieces of each such tile in workgroup order,
// so the result does not depend on timing, and runs the same epilogue.
//
// Epilogues: plain store, accumulate, fp32 split-K partials, Q/K/V with
// rotary embedding and the K/V store to pool slots, and SwiGLU.
#include <algorithm>
#include <atomic>
#include <type_traits>

#include "device.h"
#include "internal.h"

namespace acache {

namespace {

// Tile configuration.  Every wave covers 128 weight rows (one attention
// head, or 64 gate + 64 up rows) and WAVE_M activation rows.
template <int BN_, int BM_, int WN_, int WM_, int BK_>
struct Cfg {
  static constexpr int BN = BN_;       // weight rows per workgroup
  static constexpr int BM = BM_;       // activation rows per workgroup
  static constexpr int WN = WN_;       // waves along N
  static constexpr int WM = WM_;       // waves along M
  static constexpr int BK = BK_;       // K per LDS stage
  static constexpr int LDK = BK + 8;   // padded LDS row (elements)
  static constexpr int WAVES = WN * WM;
  static constexpr int THREADS = 64 * WAVES;
  static constexpr int WAVE_M = BM / WM;
  static constexpr int FM = WAVE_M / 32;  // activation fragments per wave
  static constexpr int CPR = BK / 8;      // 16-byte chunks per row
  static constexpr int W_CHUNKS = BN * CPR / THREADS;
  static constexpr int X_CHUNKS = BM * CPR / THREADS;
  static constexpr int ACC4 = 4 * FM * 4;  // float4 accumulator chunks per lane
  static_assert(BN / WN == 128, "a wave spans 128 weight rows");
  static_assert(WAVE_M % 32 == 0 && FM >= 1, "wave M extent");
  static_assert(BK % 32 == 0, "an even number of 16-wide K slices per stage");
  static_assert(BN * CPR % THREADS == 0 && BM * CPR % THREADS == 0, "load split");
};

typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4;

struct TileMap {
  int n_tiles, m_tiles;
  int splits;      // K splits (split-K partial epilogue); split i owns K steps [i nk / splits, (i+1) nk / splits)
  int nk;          // K steps of a whole tile
  int dp_rounds;   // whole tiles per workgroup, logical tile j * dp_stride + w
  int dp_stride;
  int dp_tiles;    // logical tiles of those rounds (the last round may be partial)
  int sk_first;    // first logical tile of the stream-K region
  int sk_units;    // K steps in the stream-K region
  int sk_groups;   // workgroups sharing the stream-K region (0: none)
  float* sk_part;  // [sk_groups][2][THREADS * ACC4 * 4] partial accumulators
};

constexpr int kGroupM = 4;       // M tiles per raster group
constexpr int kMaxSkGroups = 256;
constexpr int kMinSkSteps = 4;   // K steps per tile for stream-K, and per split, at least
constexpr int kMaxSplits = 16;

// Workgroups are dealt round-robin to the 8 XCDs; renumber them so that each
// XCD holds a contiguous range of logical workgroup ids.
__device__ __forceinline__ int logical_block() {
  const int nb = gridDim.x, i = blockIdx.x;
  const int q = nb >> 3, r = nb & 7;
  const int x = i & 7, slot = i >> 3;
  return x * q + min(x, r) + slot;
}

// Logical tile -> (n tile, m tile, split).  Inside a split, tiles run in
// groups of kGroupM M tiles with the M index fastest, so the workgroups
// resident at one time on an XCD share their weight tiles in its L2.
__device__ __forceinline__ void tile_coords(const TileMap& tm, int t, int& nt, int& mt, int& sp) {
  const int per_split = tm.m_tiles * tm.n_tiles;
  sp = t / per_split;
  const int u = t - sp * per_split;
  const int group = u / (kGroupM * tm.n_tiles);
  const int first_m = group * kGroupM;
  const int gm = min(tm.m_tiles - first_m, kGroupM);
  const int v = u - group * kGroupM * tm.n_tiles;
  mt = first_m + v % gm;
  nt = v / gm;
}

// Stream-K bookkeeping: workgroup w owns K steps [start(w), start(w + 1)) of
// the stream-K region; the owner of step i is the largest w with start(w) <= i.
__device__ __forceinline__ int sk_start(const TileMap& tm, int w) {
  return (int)(((int64_t)w * tm.sk_units) / tm.sk_groups);
}
__device__ __forceinline__ int sk_owner(const TileMap& tm, int i) {
  return (int)((((int64_t)i + 1) * tm.sk_groups - 1) / tm.sk_units);
}

template <int EPI, int BN>
__device__ __forceinline__ int weight_row(int nt, int r, int F) {
  if constexpr (EPI == EPI_SWIGLU) {
    // per wave half: 64 gate rows, then the matching 64 up rows
    const int half = r >> 7, w = r & 127;
    const int col = nt * (BN / 2) + half * 64 + (w & 63);
    return w < 64 ? col : F + col;
  } else {
    return nt * BN + r;
  }
}

// SiLU(gate) * up with the hardware reciprocal (about 1 ulp in fp32, far
// below the bf16 rounding of the result) instead of an IEEE division, whose
// expansion costs ten instructions per element in the epilogue.
// gate -> -inf: 1 + e^-gate = inf, reciprocal 0, result -0 (as the division).
__device__ __forceinline__ float silu_mul(float gate, float up) {
  return gate * __builtin_amdgcn_rcpf(1.f + __expf(-gate)) * up;
}

__device__ __forceinline__ void store4(bf16* p, const float v[4]) {
  bf16x4 o;
  o[0] = (bf16)v[0]; o[1] = (bf16)v[1]; o[2] = (bf16)v[2]; o[3] = (bf16)v[3];
  *reinterpret_cast<bf16x4*>(p) = o;
}

// Partial accumulators of one wave: float4 chunk i of lane l at (i * 64 + l) * 4,
// chunk i = (a * FM + b) * 4 + g holding acc[a][b][4g .. 4g + 3].
template <class C>
__device__ __forceinline__ void store_partial(float* base, const f32x16 (&acc)[4][C::FM], int lane) {
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < C::FM; ++b)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 v = {acc[a][b][4 * g], acc[a][b][4 * g + 1], acc[a][b][4 * g + 2], acc[a][b][4 * g + 3]};
        *reinterpret_cast<f32x4*>(base + (((a * C::FM + b) * 4 + g) * 64 + lane) * 4) = v;
      }
}

template <class C>
__device__ __forceinline__ void add_partial(const float* base, f32x16 (&acc)[4][C::FM], int lane) {
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < C::FM; ++b)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 v = *reinterpret_cast<const f32x4*>(base + (((a * C::FM + b) * 4 + g) * 64 + lane) * 4);
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[a][b][4 * g + j] += v[j];
      }
}

// Writes one wave's accumulators (wave (wn, wm) of tile (nt, mt), split sp).
// acc[a][b][r] = C[m = mbase + 32b + lane%32][n = nbase + 32a + 8(r/4) + 4(lane/32) + r%4]
template <int EPI, class C>
__device__ __forceinline__ void epilogue(const GemmParams& p, const f32x16 (&acc)[4][C::FM], int nt, int mt,
                                         int sp, int wn, int wm, int lane) {
  constexpr int BN = C::BN, BM = C::BM, FM = C::FM;
  const int hl = lane >> 5;
  const int mbase = mt * BM + wm * C::WAVE_M + (lane & 31);
#pragma unroll
  for (int b = 0; b < FM; ++b) {
    const int m = mbase + b * 32;
    if (m >= p.M) continue;
    if constexpr (EPI == EPI_STORE || EPI == EPI_ACCUM || EPI == EPI_PARTIAL) {
      const int nbase = nt * BN + wn * 128;
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int n = nbase + a * 32 + g * 8 + hl * 4;
          float v[4] = {acc[a][b][4 * g], acc[a][b][4 * g + 1], acc[a][b][4 * g + 2], acc[a][b][4 * g + 3]};
          if constexpr (EPI == EPI_PARTIAL) {
            float* dst = p.P + ((int64_t)sp * p.M + m) * p.N + n;
            f32x4 o = {v[0], v[1], v[2], v[3]};
            *reinterpret_cast<f32x4*>(dst) = o;
          } else {
            bf16* dst = (bf16*)p.C + (int64_t)m * p.ldc + n;
            if constexpr (EPI == EPI_ACCUM) {
              const bf16x4 old = *reinterpret_cast<const bf16x4*>(dst);
#pragma unroll
              for (int j = 0; j < 4; ++j) v[j] += (float)old[j];
            }
            store4(dst, v);
          }
        }
    } else if constexpr (EPI == EPI_SWIGLU) {
      const int cbase = nt * (BN / 2) + wn * 64;
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          float v[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float gt = acc[a][b][4 * g + j], up = acc[a + 2][b][4 * g + j];
            v[j] = silu_mul(gt, up);
          }
          store4((bf16*)p.C + (int64_t)m * p.ldc + cbase + a * 32 + g * 8 + hl * 4, v);
        }
    } else if constexpr (EPI == EPI_QKV) {
      const int col0 = nt * BN + wn * 128;  // first weight row of this wave = one head
      const bool is_v = col0 >= p.hq_cols + p.hkv_cols;
      bf16* dst;
      if (col0 < p.hq_cols) {
        dst = (bf16*)p.q_out + (int64_t)m * p.hq_cols + col0;
      } else {
        const int64_t slot = p.write_slots[m];
        if (slot < 0 || slot >= p.n_slots) continue;
        const int c = is_v ? col0 - p.hq_cols - p.hkv_cols : col0 - p.hq_cols;
        dst = (bf16*)(is_v ? p.v_pool : p.k_pool) + slot * p.pool_ld + c;
      }
      if (!is_v) {
        // rotate the pairs (d, d + 64): both halves sit in this lane, in
        // fragments a and a + 2
        const float* rt = p.rope_cs + (int64_t)m * 128;
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            float lo[4], hi[4];
            const int d0 = a * 32 + 8 * g + 4 * hl;
            const f32x4 t0 = *reinterpret_cast<const f32x4*>(rt + 2 * d0);
            const f32x4 t1 = *reinterpret_cast<const f32x4*>(rt + 2 * d0 + 4);
            const float cs4[4] = {t0[0], t0[2], t1[0], t1[2]}, sn4[4] = {t0[1], t0[3], t1[1], t1[3]};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const int r = 4 * g + j;
              const float cs = cs4[j], sn = sn4[j];
              const float x1 = acc[a][b][r], x2 = acc[a + 2][b][r];
              lo[j] = x1 * cs - x2 * sn;
              hi[j] = x2 * cs + x1 * sn;
            }
            store4(dst + a * 32 + g * 8 + hl * 4, lo);
            store4(dst + (a + 2) * 32 + g * 8 + hl * 4, hi);
          }
      } else {
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const float v[4] = {acc[a][b][4 * g], acc[a][b][4 * g + 1], acc[a][b][4 * g + 2], acc[a][b][4 * g + 3]};
            store4(dst + a * 32 + g * 8 + hl * 4, v);
          }
      }
    }
  }
}


// Main loop: a ping-pong schedule.  The K range is cut into 32-wide units.
// The waves form two groups, waves 0-3 and 4-7, one wave of each on every
// SIMD; each wave alternates a memory phase (read its MFMA fragments of the
// next unit from LDS, issue buffer -> LDS copies of the unit kAhead units
// ahead) and a compute phase (MFMAs back to back), and group 1 runs one
// phase behind group 0.  Every phase ends at a workgroup barrier, so while
// one wave of a SIMD issues matrix work the other does its memory work.  LDS
// holds a ring of kAhead + 1 units, each 256 weight rows and BM activation
// rows of 64 bytes, written by buffer_load_dwordx4 ... lds (no staging
// registers; the copies' addresses are an SGPR base and offset plus one
// fixed VGPR offset per lane); the copy of unit v + kAhead reuses the slot of
// unit v - 1, which both groups finished reading before the barrier that
// opened this phase.  Chunk c (16 B) of row r is stored at c ^ ((r >> 2) & 3)
// so that the 16 rows read by one quarter-wave hit distinct banks.  The wave
// index is made uniform so that LDS addresses and the group branches stay
// scalar.  Weights are streamed from HBM once per launch, so the depth of
// the ring is what hides HBM latency when few workgroups run.
constexpr int kPPRowB = 64;  // one 32-element unit row

// Waits until at most n units of this wave's copies (NCP each) are in flight.
template <int NCP, int MAXN>
__device__ __forceinline__ void wait_units(int n) {
  if constexpr (MAXN == 0) {
    wait_vmcnt<0>();
  } else {
    if (n >= MAXN) wait_vmcnt<NCP * MAXN>();
    else wait_units<NCP, MAXN - 1>(n);
  }
}

template <int EPI, class C>
__global__ __launch_bounds__(C::THREADS) void gemm_bf16_kernel(GemmParams p, TileMap tm) {
  static_assert(C::BN == 256 && (C::BM == 256 || C::BM == 128) && C::WN == 2 && C::WM == 4 && C::BK == 64,
                "ping-pong tile");
  constexpr int FM = C::FM;
  constexpr int XI = C::BM / 128;               // activation copies per wave and unit
  constexpr int NCP = 2 + XI;                   // copies per wave and unit
  constexpr int kStageB = (256 + C::BM) * kPPRowB;
  // ring depth: copies run kAhead units ahead of the fragment reads (deeper
  // rings measured slower, also with weights streamed from HBM)
  constexpr int kStages = 4;
  constexpr int kAhead = kStages - 1;
  __shared__ __attribute__((aligned(1024))) char ring[kStages * kStageB];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: LDS addresses in SGPRs
  const int wn = wave % C::WN, wm = wave / C::WN;
  const int grp = wave >> 2;
  const int F = p.N >> 1;
  const bf16* __restrict__ X = (const bf16*)p.X;
  const bf16* __restrict__ W = (const bf16*)p.W;
  const int K = p.K;
  const int nk_tile = tm.nk;
  const int w = logical_block();

  // copies: wave v fills weight rows [32 v, 32 v + 32) and activation rows
  // [16 XI v, 16 XI v + 16 XI), 16 rows per instruction; lane l takes row
  // 16 i + l / 4 and physical chunk l % 4
  const int crow = lane >> 2;
  const int cchunk = (lane & 3) ^ ((lane >> 4) & 3);
  // fragment reads: row (lane % 32) of each 32-row fragment; the swizzle
  // of every such row is ((lane % 32) >> 2) & 3
  const int fsw = ((lane & 31) >> 2) & 3;
  const int arow = wn * 128 + (lane & 31);
  const int brow = 256 + wm * C::WAVE_M + (lane & 31);
  const int cofs0 = ((0 + (lane >> 5)) ^ fsw) * 16;  // slice 0: chunks 0 / 1
  const int cofs1 = ((2 + (lane >> 5)) ^ fsw) * 16;  // slice 1: chunks 2 / 3
  const __amdgpu_buffer_rsrc_t wres = buffer_rsrc(W, (uint32_t)p.N * (uint32_t)K * 2u);
  const __amdgpu_buffer_rsrc_t xres = buffer_rsrc(X, (uint32_t)p.M * (uint32_t)K * 2u);

  f32x16 acc[4][FM];
  int item = 0;
  int u = 0, u_end = 0;
  if (tm.sk_groups > 0 && w < tm.sk_groups) {
    u = sk_start(tm, w);
    u_end = sk_start(tm, w + 1);
  }
  int piece = 0;
  while (true) {
    int t, kb, kn;
    bool sk = false;
    if (item < tm.dp_rounds) {
      t = item * tm.dp_stride + w;
      if (t >= tm.dp_tiles) break;
      kb = -1;
      kn = 0;
      ++item;
    } else if (u < u_end) {
      const int tl = u / nk_tile;
      kb = u - tl * nk_tile;
      kn = min(nk_tile - kb, u_end - u);
      t = tm.sk_first + tl;
      u += kn;
      sk = true;
    } else {
      break;
    }
    int nt, mt, sp;
    tile_coords(tm, t, nt, mt, sp);
    if (kb < 0) {
      kb = sp * nk_tile / tm.splits;
      kn = (sp + 1) * nk_tile / tm.splits - kb;
    }
    const int k0 = kb * C::BK;
    const int U = 2 * kn;  // 32-wide units

    // byte offsets from the uniform base pointers (operands stay below 2^31
    // elements), so the copies use the SGPR-base + 32-bit offset form
    uint32_t wsrc[2], xsrc[XI];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int r = wave * 32 + i * 16 + crow;
      wsrc[i] = (uint32_t)(weight_row<EPI, 256>(nt, r, F) * K + k0 + cchunk * 8) * 2u;
    }
#pragma unroll
    for (int i = 0; i < XI; ++i) {
      const int r = wave * 16 * XI + i * 16 + crow;
      xsrc[i] = (uint32_t)(min(mt * C::BM + r, p.M - 1) * K + k0 + cchunk * 8) * 2u;
    }
    auto issue = [&](int v) {
      char* st = ring + (v % kStages) * kStageB;
      const uint32_t ko = (uint32_t)v * 64u;  // uniform: the SGPR offset of the buffer loads
#pragma unroll
      for (int i = 0; i < 2; ++i) dma16_buf(wres, wsrc[i], ko, st + (wave * 32 + i * 16) * kPPRowB);
#pragma unroll
      for (int i = 0; i < XI; ++i) dma16_buf(xres, xsrc[i], ko, st + (256 + wave * 16 * XI + i * 16) * kPPRowB);
    };
    bf16x8 af[2][4], bfr[2][FM];
    auto read_frags = [&](int v) {
      const char* st = ring + (v % kStages) * kStageB;
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        af[0][a] = *reinterpret_cast<const bf16x8*>(st + (arow + a * 32) * kPPRowB + cofs0);
        af[1][a] = *reinterpret_cast<const bf16x8*>(st + (arow + a * 32) * kPPRowB + cofs1);
      }
#pragma unroll
      for (int b = 0; b < FM; ++b) {
        bfr[0][b] = *reinterpret_cast<const bf16x8*>(st + (brow + b * 32) * kPPRowB + cofs0);
        bfr[1][b] = *reinterpret_cast<const bf16x8*>(st + (brow + b * 32) * kPPRowB + cofs1);
      }
    };

#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < FM; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;

    // the previous item's stores and copies are complete, and every wave is
    // past its last LDS read of the previous item
    wait_vmcnt<0>();
    lds_barrier();
#pragma unroll
    for (int v = 0; v < kAhead; ++v)
      if (v < U) issue(v);
    wait_units<NCP, kAhead - 1>(min(U, kAhead) - 1);  // unit 0 is in LDS
    bare_barrier();
    if (grp == 1) bare_barrier();  // group 1 runs one phase behind
    for (int v = 0; v < U; ++v) {
      // memory phase
      __builtin_amdgcn_sched_barrier(0);
      read_frags(v);
      if (v + kAhead < U) issue(v + kAhead);
      // this wave's copies of unit v + 1 are complete before the barrier
      if (v + 1 < U) wait_units<NCP, kAhead - 1>(min(U - 1, v + kAhead) - (v + 1));
      wait_lgkmcnt<0>();
      __builtin_amdgcn_sched_barrier(0);
      bare_barrier();
      __builtin_amdgcn_sched_barrier(0);
      // compute phase
#pragma unroll
      for (int s = 0; s < 2; ++s)
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
          for (int b = 0; b < FM; ++b) acc[a][b] = mfma32x32x16(af[s][a], bfr[s][b], acc[a][b]);
      __builtin_amdgcn_sched_barrier(0);
      bare_barrier();
    }
    if (grp == 0) bare_barrier();  // the phase in which group 1 computes the last unit

    if (sk && kn < nk_tile) {
      float* slot = tm.sk_part + ((size_t)(w * 2 + piece) * C::WAVES + wave) * (64 * C::ACC4 * 4);
      store_partial<C>(slot, acc, lane);
      ++piece;
    } else {
      if (sk) ++piece;
      epilogue<EPI, C>(p, acc, nt, mt, sp, wn, wm, lane);
    }
  }
}

// ---------------------------------------------------------------------------
// 16x16x32 MFMA tiles (gfx950 issues them at a higher rate than 32x32x16:
// measured 86% against 69% of the bf16 peak for back-to-back independent
// MFMAs from one wave per SIMD).  Lane l supplies A[l % 16][8 (l / 16) + j]
// and B[8 (l / 16) + j][l % 16], j = 0..7, and receives
// D[4 (l / 16) + r][l % 16] in accumulator register r = 0..3.  With the
// weights as A, lane l holds activation row l % 16 and output columns
// 4 (l / 16) .. + 3 of each 16 x 16 tile.
// The accumulator is held in AGPRs by the asm constraint
// (the compiler otherwise moves a 256-register accumulator set between
// AGPRs and VGPRs on every loop iteration).  The hazard recognizer does not
// look into inline asm: callers pad with s_nop where the accumulators pass
// between VALU and MFMA (mfma_agpr_fence).
__device__ __forceinline__ void mfma16x16x32_agpr(f32x4& c, bf16x8 a, bf16x8 b) {
  asm("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(c) : "v"(a), "v"(b));
}
// Wait states between MFMA results in AGPRs and their VALU readers (or
// VALU-written AGPRs and a following MFMA), more than any gfx950 MFMA needs.
__device__ __forceinline__ void mfma_agpr_fence() { asm volatile("s_nop 7\n s_nop 7\n s_nop 7" ::: "memory"); }

// One wave's 128 x 128 accumulators: acc[a][b][r] = C[m = mbase + 16 b + lane % 16]
// [n = nbase + 16 a + 4 (lane / 16) + r].
typedef f32x4 Acc16[8][8];

// Partial accumulators: float4 chunk i = a * 8 + b of lane l at (i * 64 + l) * 4.
__device__ __forceinline__ void store_partial16(float* base, const Acc16& acc, int lane) {
#pragma unroll
  for (int a = 0; a < 8; ++a)
#pragma unroll
    for (int b = 0; b < 8; ++b) *reinterpret_cast<f32x4*>(base + ((a * 8 + b) * 64 + lane) * 4) = acc[a][b];
}

// Writes one wave's accumulators (wave (wn, wm) of 256 x 256 tile (nt, mt),
// split sp): the same epilogues as the 32x32 layout.  acc[a][bb] holds the
// 16-row block b = B0 + bb (NB of the wave's 8).
template <int EPI, int B0 = 0, int NB = 8>
__device__ __forceinline__ void epilogue16(const GemmParams& p, const f32x4 (&acc)[8][NB], int nt, int mt, int sp,
                                           int wn, int wm, int lane) {
  // lane-dependent addresses are computed here, per item: hoisted out of the
  // item loop they would be held through the K loop and spilled
  lane = lane_id_here();
  const int q4 = 4 * (lane >> 4);
  const int mbase = mt * 256 + wm * 128 + (lane & 15);
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const int m = mbase + (B0 + b) * 16;
    if (m >= p.M) continue;
    if constexpr (EPI == EPI_STORE || EPI == EPI_ACCUM || EPI == EPI_PARTIAL) {
      const int nbase = nt * 256 + wn * 128 + q4;
#pragma unroll
      for (int a = 0; a < 8; ++a) {
        const int n = nbase + a * 16;
        float v[4] = {acc[a][b][0], acc[a][b][1], acc[a][b][2], acc[a][b][3]};
        if constexpr (EPI == EPI_PARTIAL) {
          *reinterpret_cast<f32x4*>(p.P + ((int64_t)sp * p.M + m) * p.N + n) = acc[a][b];
        } else {
          bf16* dst = (bf16*)p.C + (int64_t)m * p.ldc + n;
          if constexpr (EPI == EPI_ACCUM) {
            const bf16x4 old = *reinterpret_cast<const bf16x4*>(dst);
#pragma unroll
            for (int j = 0; j < 4; ++j) v[j] += (float)old[j];
          }
          store4(dst, v);
        }
      }
    } else if constexpr (EPI == EPI_SWIGLU) {
      // tiles 0..3 of the wave are gate rows, 4..7 the matching up rows
      const int cbase = nt * 128 + wn * 64 + q4;
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        float v[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float gt = acc[a][b][j], up = acc[a + 4][b][j];
          v[j] = silu_mul(gt, up);
        }
        store4((bf16*)p.C + (int64_t)m * p.ldc + cbase + a * 16, v);
      }
    } else if constexpr (EPI == EPI_QKV) {
      const int col0 = nt * 256 + wn * 128;  // first weight row of this wave = one head
      const bool is_v = col0 >= p.hq_cols + p.hkv_cols;
      bf16* dst;
      if (col0 < p.hq_cols) {
        dst = (bf16*)p.q_out + (int64_t)m * p.hq_cols + col0;
      } else {
        const int64_t slot = p.write_slots[m];
        if (slot < 0 || slot >= p.n_slots) continue;
        const int c = is_v ? col0 - p.hq_cols - p.hkv_cols : col0 - p.hq_cols;
        dst = (bf16*)(is_v ? p.v_pool : p.k_pool) + slot * p.pool_ld + c;
      }
      if (!is_v) {
        // rotate the pairs (d, d + 64): both halves sit in this lane, in
        // tiles a and a + 4
        const float* rt = p.rope_cs + (int64_t)m * 128;
#pragma unroll
        for (int a = 0; a < 4; ++a) {
          float lo[4], hi[4];
          const int d0 = a * 16 + q4;
          const f32x4 t0 = *reinterpret_cast<const f32x4*>(rt + 2 * d0);
          const f32x4 t1 = *reinterpret_cast<const f32x4*>(rt + 2 * d0 + 4);
          const float cs4[4] = {t0[0], t0[2], t1[0], t1[2]}, sn4[4] = {t0[1], t0[3], t1[1], t1[3]};
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float cs = cs4[j], sn = sn4[j];
            const float x1 = acc[a][b][j], x2 = acc[a + 4][b][j];
            lo[j] = x1 * cs - x2 * sn;
            hi[j] = x2 * cs + x1 * sn;
          }
          store4(dst + a * 16 + q4, lo);
          store4(dst + (a + 4) * 16 + q4, hi);
        }
      } else {
#pragma unroll
        for (int a = 0; a < 8; ++a) {
          const float v[4] = {acc[a][b][0], acc[a][b][1], acc[a][b][2], acc[a][b][3]};
          store4(dst + a * 16 + q4, v);
        }
      }
    }
  }
}

// Main loop with one wave per SIMD: 4 waves (2 along N x 2 along M), each a
// 128 x 128 wave tile = 8 x 8 MFMA 16x16x32 tiles, 256 fp32 accumulators
// per lane (0.5 KB of LDS fragment reads per 32 x 32 x 16 of work).
//
// LDS holds the 256 weight rows of three 64-wide K steps and the 256
// activation rows of two, rows of 128 bytes (160 KB in all).  Each copy
// instruction moves 8 whole rows (a 128-byte line per row, so every L2
// request is a full line), buffer -> LDS with no staging registers.  16-byte
// chunk c of row r sits at c ^ ((r >> 1) & 7): the 16 rows read by one
// 16-lane pass of a fragment read hit 16 distinct bank groups.  The MFMAs
// run in 32-wide units, two per step.  Before unit u each wave waits for its
// fragment reads of unit u and meets the others at a barrier; it then reads
// unit u + 1's 16 fragments into the other register set, one read after
// every third of unit u's first 46 MFMAs (the last read then has 18 MFMAs
// to land before the unit's wait).  Unit 0 of step j sends step j + 2's
// weight rows into the weight stage of step j - 1 (every wave was done with
// it at the barrier before unit 1 of step j - 1), unit 1 its activation rows
// into step j's activation stage, one copy after every eighth MFMA: the L2 ->
// LDS path carries the same load in both units, and step j + 1 is complete
// once no more than step j + 2's weight copies are in flight.
constexpr int kW4RowB = 128;
constexpr int kW4StageB = 256 * kW4RowB;  // one operand's rows of one K step

template <int EPI, class C>
__global__ __launch_bounds__(C::THREADS, 1) void gemm_bf16_w4_kernel(GemmParams p, TileMap tm) {
  static_assert(C::BN == 256 && C::BM == 256 && C::WN == 2 && C::WM == 2 && C::BK == 64, "4-wave tile");
  // weight stages 0..2, then activation stages 0..1
  __shared__ __attribute__((aligned(1024))) char ring[5 * kW4StageB];
  char* const xring = ring + 3 * kW4StageB;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wn = wave & 1, wm = wave >> 1;
  const int F = p.N >> 1;
  const int K = p.K;
  const int nk_tile = tm.nk;
  const int w = logical_block();

  // copies: instruction i of a wave covers rows 64 wave + 8 i + lane / 8;
  // the lane fills physical chunk lane % 8 with logical chunk
  // (lane % 8) ^ ((row >> 1) & 7)
  const int crow = lane >> 3;
  // fragment reads: row lane % 16 of each 16-row fragment, chunk 4 h + lane / 16
  const int fsw = ((lane & 15) >> 1) & 7;
  const int arow = wn * 128 + (lane & 15);
  const int brow = wm * 128 + (lane & 15);
  const int cofs0 = ((0 + (lane >> 4)) ^ fsw) * 16;
  const int cofs1 = ((4 + (lane >> 4)) ^ fsw) * 16;
  const __amdgpu_buffer_rsrc_t wres = buffer_rsrc(p.W, (uint32_t)p.N * (uint32_t)K * 2u);
  const __amdgpu_buffer_rsrc_t xres = buffer_rsrc(p.X, (uint32_t)p.M * (uint32_t)K * 2u);

  Acc16 acc;
  int item = 0;
  int u = 0, u_end = 0;
  if (tm.sk_groups > 0 && w < tm.sk_groups) {
    u = sk_start(tm, w);
    u_end = sk_start(tm, w + 1);
  }
  int piece = 0;
  while (true) {
    int t, kb, kn;
    bool sk = false;
    if (item < tm.dp_rounds) {
      t = item * tm.dp_stride + w;
      if (t >= tm.dp_tiles) break;
      kb = -1;
      kn = 0;
      ++item;
    } else if (u < u_end) {
      const int tl = u / nk_tile;
      kb = u - tl * nk_tile;
      kn = min(nk_tile - kb, u_end - u);
      t = tm.sk_first + tl;
      u += kn;
      sk = true;
    } else {
      break;
    }
    int nt, mt, sp;
    tile_coords(tm, t, nt, mt, sp);
    if (kb < 0) {
      kb = sp * nk_tile / tm.splits;
      kn = (sp + 1) * nk_tile / tm.splits - kb;
    }
    const int k0 = kb * C::BK;

    // the lane's copy offsets are recomputed per item from a lane index the
    // compiler cannot hoist: hoisted out of the item loop they are held
    // through the K loop, spilled, and reloaded one wait at a time
    const int ln = lane_id_here();
    uint32_t wsrc[8], xsrc[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int r = wave * 64 + i * 8 + (ln >> 3);
      const int c = (ln & 7) ^ ((4 * i + (ln >> 4)) & 7);
      wsrc[i] = (uint32_t)(weight_row<EPI, 256>(nt, r, F) * K + k0 + c * 8) * 2u;
      xsrc[i] = (uint32_t)(min(mt * C::BM + r, p.M - 1) * K + k0 + c * 8) * 2u;
    }
    // copy i (0..7) of K step j: 8 weight rows into weight stage j % 3, or
    // 8 activation rows into activation stage j % 2
    auto copy_w = [&](int j, int i) {
      dma16_buf(wres, wsrc[i], (uint32_t)j * 128u, ring + (j % 3) * kW4StageB + (wave * 64 + i * 8) * kW4RowB);
    };
    auto copy_x = [&](int j, int i) {
      dma16_buf(xres, xsrc[i], (uint32_t)j * 128u, xring + (j & 1) * kW4StageB + (wave * 64 + i * 8) * kW4RowB);
    };
    auto issue = [&](int j) {
#pragma unroll
      for (int i = 0; i < 8; ++i) copy_w(j, i);
#pragma unroll
      for (int i = 0; i < 8; ++i) copy_x(j, i);
    };
    // fragment f of unit h (0 / 1) of step j: f < 8 weight tile f, else
    // activation tile f - 8
    auto frag = [&](int j, int h, int f) {
      const char* st = f < 8 ? ring + (j % 3) * kW4StageB : xring + (j & 1) * kW4StageB;
      const int row = f < 8 ? arow + f * 16 : brow + (f - 8) * 16;
      return *reinterpret_cast<const bf16x8*>(st + row * kW4RowB + (h ? cofs1 : cofs0));
    };

#pragma unroll
    for (int a = 0; a < 8; ++a)
#pragma unroll
      for (int b = 0; b < 8; ++b)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[a][b][r] = 0.f;

    // every wave is past its last LDS read of the previous item (the copies
    // of the previous item have landed before its epilogue).  Its stores need
    // not drain before these copies go out: loads complete in issue order, so
    // the wait for step 0 below holds however the stores complete, and the
    // copies' latency overlaps the stores' drain.
    lds_barrier();
    issue(0);
    if (kn > 1) {
      issue(1);
      wait_vmcnt<16>();  // step 0 (this wave's part)
    } else {
      wait_vmcnt<0>();
    }
    __builtin_amdgcn_sched_barrier(0);
    bare_barrier();
    __builtin_amdgcn_sched_barrier(0);
    bf16x8 fx[16], fy[16];
#pragma unroll
    for (int f = 0; f < 16; ++f) fx[f] = frag(0, 0, f);
    mfma_agpr_fence();  // the zeroed accumulators before the first MFMA

    // 64 MFMAs from cur, the 16 reads of the next unit into nxt among the
    // first 46,
    // and (copies) the 8 weight (CX false) or activation (CX true) copies of
    // K step cj, one after every eighth MFMA (a burst of copies stalls the
    // wave's MFMA issue while the memory pipeline takes them)
    auto unit = [&](bf16x8 (&cur)[16], bf16x8 (&nxt)[16], int nj, int nh, int cj, auto cx, auto copies) {
#pragma unroll
      for (int i = 0; i < 64; ++i) {
        const int a = i >> 3, b = i & 7;
        if constexpr (decltype(copies)::value) {
          if ((i & 7) == 3) {
            if constexpr (decltype(cx)::value) copy_x(cj, i >> 3);
            else copy_w(cj, i >> 3);
          }
        }
        if (i % 3 == 0 && i / 3 < 16) nxt[i / 3] = frag(nj, nh, i / 3);
        mfma16x16x32_agpr(acc[a][b], cur[a], cur[8 + b]);
        __builtin_amdgcn_sched_barrier(0);
      }
    };
    // K step j with (copies) the copies of step j + 2
    auto step = [&](int j, auto copies) {
      constexpr bool CP = decltype(copies)::value;
      // unit 0 of step j: the weight stage of step j - 1 is free (every wave
      // passed the barrier before unit 1 of step j - 1 after its last read)
      wait_lgkmcnt<0>();
      __builtin_amdgcn_sched_barrier(0);
      bare_barrier();
      __builtin_amdgcn_sched_barrier(0);
      unit(fx, fy, j, 1, j + 2, std::false_type(), copies);
      // unit 1 of step j: step j + 1 complete in every wave (copies complete
      // in issue order: in flight after it only step j + 2's weight rows),
      // step j's activation stage free for step j + 2's
      wait_vmcnt<CP ? 8 : 0>();
      wait_lgkmcnt<0>();
      __builtin_amdgcn_sched_barrier(0);
      bare_barrier();
      __builtin_amdgcn_sched_barrier(0);
      // after the last step this reads step j's own stage (complete, not
      // written any more); the values are not used
      unit(fy, fx, j + 1 < kn ? j + 1 : j, 0, j + 2, std::true_type(), copies);
      // every step ends with the MFMA results landed: the compiler may place
      // register copies or spill code of the accumulators on any loop edge
      // (the exit of the first loop below among them), and inline asm
      // hides the MFMAs from its hazard recognizer.  The wait overlaps the
      // last MFMAs' own pipeline occupancy (measured cost under 1%).
      mfma_agpr_fence();
    };
    int j = 0;
    for (; j + 2 < kn; ++j) step(j, std::true_type());
    for (; j < kn; ++j) step(j, std::false_type());
    // every wave is past its last read of the ring, and every copy has landed
    wait_vmcnt<0>();
    lds_barrier();

    if (sk && kn < nk_tile) {
      float* slot = tm.sk_part + ((size_t)(w * 2 + piece) * C::WAVES + wave) * (64 * 256);
      store_partial16(slot, acc, lane);
      ++piece;
    } else {
      if (sk) ++piece;
      epilogue16<EPI>(p, acc, nt, mt, sp, wn, wm, lane);
    }
  }
}

// Stream-K fixup of the 16x16 tiles: block = one wave-tile of one split
// tile of the stream-K region; its wave q sums the rows 32 q .. 32 q + 31 of
// the tile's pieces in workgroup order and runs their epilogue.
template <int EPI, class C>
__global__ __launch_bounds__(256) void gemm_bf16_fixup16(GemmParams p, TileMap tm) {
  constexpr int kPieceF = 64 * 256;  // floats per wave piece
  const int tid = threadIdx.x, lane = tid & 63;
  const int q = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int s = blockIdx.x / C::WAVES, wave = blockIdx.x % C::WAVES;
  const int wn = wave & 1, wm = wave >> 1;
  const int nk_tile = tm.nk;
  const int first = sk_owner(tm, s * nk_tile), last = sk_owner(tm, (s + 1) * nk_tile - 1);
  if (first == last) return;  // the tile was finished by one workgroup
  int nt, mt, sp;
  tile_coords(tm, tm.sk_first + s, nt, mt, sp);
  auto run = [&](auto qc) {
    constexpr int Q = decltype(qc)::value;
    f32x4 acc[8][2];
#pragma unroll
    for (int a = 0; a < 8; ++a)
#pragma unroll
      for (int bb = 0; bb < 2; ++bb)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[a][bb][r] = 0.f;
#pragma unroll 2
    for (int w = first; w <= last; ++w) {
      // piece 0 of w if w's range starts in this tile, else its piece 1
      const int pc = sk_start(tm, w) / nk_tile == s ? 0 : 1;
      const float* src = tm.sk_part + ((size_t)(w * 2 + pc) * C::WAVES + wave) * kPieceF;
      f32x4 v[8][2];
#pragma unroll
      for (int a = 0; a < 8; ++a)
#pragma unroll
        for (int bb = 0; bb < 2; ++bb)
          v[a][bb] = *reinterpret_cast<const f32x4*>(src + ((a * 8 + 2 * Q + bb) * 64 + lane) * 4);
#pragma unroll
      for (int a = 0; a < 8; ++a)
#pragma unroll
        for (int bb = 0; bb < 2; ++bb)
#pragma unroll
          for (int r = 0; r < 4; ++r) acc[a][bb][r] += v[a][bb][r];
    }
    epilogue16<EPI, 2 * Q, 2>(p, acc, nt, mt, sp, wn, wm, lane);
  };
  switch (q) {
    case 0: run(std::integral_constant<int, 0>()); break;
    case 1: run(std::integral_constant<int, 1>()); break;
    case 2: run(std::integral_constant<int, 2>()); break;
    default: run(std::integral_constant<int, 3>()); break;
  }
}

// Stream-K fixup: block = one wave-tile of one split tile of the stream-K
// region.  Sums the tile's pieces in workgroup order and runs the epilogue.
// The pieces are read four at a time: wave 0 adds the first of a round from
// memory while waves 1-3 copy the next three to LDS, then wave 0 adds those
// in order, so the sum is p_first + p_first+1 + ... as one sequential loop.
template <int EPI, class C>
__global__ __launch_bounds__(256) void gemm_bf16_fixup(GemmParams p, TileMap tm) {
  constexpr int kPieceF = 64 * C::ACC4 * 4;  // floats per wave piece
  // pieces staged per round: three of a 128 x 64 wave tile, two of a 128 x 128 one
  constexpr int kDepth = 3 * kPieceF * 4 <= 128 * 1024 ? 3 : 2;
  __shared__ __attribute__((aligned(16))) float stage[kDepth][kPieceF];
  const int tid = threadIdx.x, lane = tid & 63;
  const int q = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int s = blockIdx.x / C::WAVES, wave = blockIdx.x % C::WAVES;
  const int wn = wave % C::WN, wm = wave / C::WN;
  const int nk_tile = tm.nk;
  const int first = sk_owner(tm, s * nk_tile), last = sk_owner(tm, (s + 1) * nk_tile - 1);
  if (first == last) return;  // the tile was finished by one workgroup
  // piece 0 of w if w's range starts in this tile, else its piece 1
  auto piece = [&](int w) {
    const int pc = sk_start(tm, w) / nk_tile == s ? 0 : 1;
    return tm.sk_part + ((size_t)(w * 2 + pc) * C::WAVES + wave) * kPieceF;
  };
  f32x16 acc[4][C::FM];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < C::FM; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;
  for (int w0 = first; w0 <= last; w0 += kDepth + 1) {
    if (q > 0 && q <= kDepth && w0 + q <= last) {
      const float* src = piece(w0 + q);
      float* dst = stage[q - 1];
#pragma unroll 8
      for (int i = 0; i < C::ACC4; ++i)
        *reinterpret_cast<f32x4*>(dst + (i * 64 + lane) * 4) =
            *reinterpret_cast<const f32x4*>(src + (i * 64 + lane) * 4);
    }
    if (q == 0) add_partial<C>(piece(w0), acc, lane);
    __syncthreads();
    if (q == 0) {
      for (int j = 1; j <= kDepth && w0 + j <= last; ++j) add_partial<C>(stage[j - 1], acc, lane);
    }
    __syncthreads();
  }
  if (q != 0) return;
  int nt, mt, sp;
  tile_coords(tm, tm.sk_first + s, nt, mt, sp);
  epilogue<EPI, C>(p, acc, nt, mt, sp, wn, wm, lane);
}

}  // namespace

// The 256 x 128 tile (8 waves, 1.25 KB of LDS reads per 32x32x16 MFMA)
// doubles the tile count for row counts that would leave CUs idle.
// 256 x 256 tiles: 4 waves of 128 x 128 on 16x16x32 MFMAs (gemm_bf16_w4_kernel);
// 256 x 128 tiles: the 8-wave ping-pong kernel on 32x32x16 MFMAs
using GemmCfg = Cfg<256, 256, 2, 2, 64>;
using GemmCfgH = Cfg<256, 128, 2, 4, 64>;

namespace {

// Time of one K step of a 256 x 128 tile relative to one of a 256 x 256 tile
// at the same number of busy CUs (measured 0.65 - 0.71: the half tile reads
// more LDS bytes per MFMA).
constexpr double kHalfStep = 0.7;

int cu_count() {
  static std::atomic<int> cached[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return kMaxSkGroups;
  int n = cached[dev].load(std::memory_order_relaxed);
  if (n == 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = kMaxSkGroups;
    cached[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

template <class C>
constexpr double step_cost() {
  return C::BM == 256 ? 1.0 : kHalfStep;
}

// K splits for the split-K partial epilogue, and their cost in 256 x 256 K
// steps of one workgroup, on kMaxSkGroups CUs (fixed, so the workspace plan
// and the launch agree on any device): ceil(T s / G) rounds of ceil(nk / s)
// steps, plus s fp32 slices of M x N written here and read back by the
// reduction, about M N 8 / 9.5e6 K steps each at HBM speed.  Splits need not
// divide nk; each keeps at least kMinSkSteps steps.
template <class C>
int splits_for(int M, int N, int K, double* cost_out) {
  const int tiles = ((M + C::BM - 1) / C::BM) * (N / C::BN);
  const int nk = K / C::BK;
  const int G = kMaxSkGroups;
  const double slice = (double)M * N * 8.0 / 9.5e6;
  int best = 1;
  double best_cost = 1e30;
  for (int s = 1; s <= kMaxSplits && nk / s >= kMinSkSteps; ++s) {
    const double cost =
        (double)((tiles * s + G - 1) / G) * ((nk + s - 1) / s) * step_cost<C>() + s * slice;
    if (cost < best_cost) {
      best_cost = cost;
      best = s;
    }
  }
  if (cost_out) *cost_out = best_cost;
  return best;
}

// The split-K epilogue's tile: a function of the shape only, so that the
// caller's split count (which sizes its partial buffer) and the launch agree.
bool partial_half(int M, int N, int K) {
  double c256 = 0, c128 = 0;
  splits_for<GemmCfg>(M, N, K, &c256);
  splits_for<GemmCfgH>(M, N, K, &c128);
  return c128 < c256;
}

struct Plan {
  TileMap tm;
  int grid;
  int sk_tiles;
  double cost;  // in 256 x 256 K steps of one workgroup
};

template <class C>
Plan plan_cfg(GemmEpi epi, const GemmParams& p) {
  Plan pl = {};
  TileMap& tm = pl.tm;
  tm.m_tiles = (p.M + C::BM - 1) / C::BM;
  tm.n_tiles = epi == EPI_SWIGLU ? (p.N / 2) / (C::BN / 2) : p.N / C::BN;
  tm.splits = epi == EPI_PARTIAL ? p.splits : 1;
  tm.nk = p.K / C::BK;
  const int tiles = tm.m_tiles * tm.n_tiles * tm.splits;
  const int nk = tm.nk;
  const int G = std::min(cu_count(), kMaxSkGroups);
  pl.grid = tiles;
  tm.dp_rounds = 1;
  tm.dp_stride = tiles;
  tm.dp_tiles = tiles;
  const double dp_cost = (double)((tiles + G - 1) / G) * ((nk + tm.splits - 1) / tm.splits);
  double best = dp_cost;
  if (epi != EPI_PARTIAL && p.sk_ws && nk >= kMinSkSteps) {
    // Stream-K with g workgroups on the e tiles left after r full rounds:
    // r whole tiles, ceil(e nk / g) steps, and the partial pieces (at most
    // e + g, each written and read back once), which cost about 1/8 of a K
    // step each (measured).  With g >= e every range spans at most nk steps
    // and so touches at most two tiles (the two partial slots of a
    // workgroup).
    const int r = tiles / G, e = tiles % G;
    int best_g = 0;
    for (int g = e; e > 0 && g <= G; ++g) {
      const double cost = (double)r * nk + (double)((e * nk + g - 1) / g) + (e + g) / 8.0;
      if (cost < best) {
        best = cost;
        best_g = g;
      }
    }
    if (best_g > 0) {
      tm.dp_rounds = r;
      tm.dp_stride = G;
      tm.dp_tiles = r * G;
      tm.sk_first = r * G;
      tm.sk_units = e * nk;
      tm.sk_groups = best_g;
      tm.sk_part = p.sk_ws;
      pl.grid = r > 0 ? G : best_g;
      pl.sk_tiles = e;
    }
  }
  if (pl.sk_tiles == 0 && tiles > G && tiles % G != 0) {
    // data-parallel rounds ending in a partial one run on G persistent
    // workgroups, a workgroup's next tile starting its copies while the last
    // one's stores drain (measured at 68,800 rows: QKV 4% and down 3% faster;
    // on whole rounds, gate/up at 278,528 rows, 2% slower, so those keep one
    // workgroup per tile)
    tm.dp_rounds = (tiles + G - 1) / G;
    tm.dp_stride = G;
    pl.grid = G;
  }
  pl.cost = best * step_cost<C>();
  return pl;
}

template <class C>
hipError_t launch_plan(GemmEpi epi, const GemmParams& p, const Plan& pl, hipStream_t s) {
  const TileMap& tm = pl.tm;
  const dim3 grid(pl.grid), block(C::THREADS);
  if constexpr (C::WAVES == 4) {
    switch (epi) {
      case EPI_STORE: hipLaunchKernelGGL((gemm_bf16_w4_kernel<EPI_STORE, C>), grid, block, 0, s, p, tm); break;
      case EPI_ACCUM: hipLaunchKernelGGL((gemm_bf16_w4_kernel<EPI_ACCUM, C>), grid, block, 0, s, p, tm); break;
      case EPI_PARTIAL: hipLaunchKernelGGL((gemm_bf16_w4_kernel<EPI_PARTIAL, C>), grid, block, 0, s, p, tm); break;
      case EPI_QKV: hipLaunchKernelGGL((gemm_bf16_w4_kernel<EPI_QKV, C>), grid, block, 0, s, p, tm); break;
      case EPI_SWIGLU: hipLaunchKernelGGL((gemm_bf16_w4_kernel<EPI_SWIGLU, C>), grid, block, 0, s, p, tm); break;
    }
  } else {
    switch (epi) {
      case EPI_STORE: hipLaunchKernelGGL((gemm_bf16_kernel<EPI_STORE, C>), grid, block, 0, s, p, tm); break;
      case EPI_ACCUM: hipLaunchKernelGGL((gemm_bf16_kernel<EPI_ACCUM, C>), grid, block, 0, s, p, tm); break;
      case EPI_PARTIAL: hipLaunchKernelGGL((gemm_bf16_kernel<EPI_PARTIAL, C>), grid, block, 0, s, p, tm); break;
      case EPI_QKV: hipLaunchKernelGGL((gemm_bf16_kernel<EPI_QKV, C>), grid, block, 0, s, p, tm); break;
      case EPI_SWIGLU: hipLaunchKernelGGL((gemm_bf16_kernel<EPI_SWIGLU, C>), grid, block, 0, s, p, tm); break;
    }
  }
  if (pl.sk_tiles > 0) {
    const dim3 fgrid(pl.sk_tiles * C::WAVES), fblock(256);
    if constexpr (C::WAVES == 4) {
      switch (epi) {
        case EPI_STORE: hipLaunchKernelGGL((gemm_bf16_fixup16<EPI_STORE, C>), fgrid, fblock, 0, s, p, tm); break;
        case EPI_ACCUM: hipLaunchKernelGGL((gemm_bf16_fixup16<EPI_ACCUM, C>), fgrid, fblock, 0, s, p, tm); break;
        case EPI_QKV: hipLaunchKernelGGL((gemm_bf16_fixup16<EPI_QKV, C>), fgrid, fblock, 0, s, p, tm); break;
        case EPI_SWIGLU: hipLaunchKernelGGL((gemm_bf16_fixup16<EPI_SWIGLU, C>), fgrid, fblock, 0, s, p, tm); break;
        default: break;
      }
    } else {
      switch (epi) {
        case EPI_STORE: hipLaunchKernelGGL((gemm_bf16_fixup<EPI_STORE, C>), fgrid, fblock, 0, s, p, tm); break;
        case EPI_ACCUM: hipLaunchKernelGGL((gemm_bf16_fixup<EPI_ACCUM, C>), fgrid, fblock, 0, s, p, tm); break;
        case EPI_QKV: hipLaunchKernelGGL((gemm_bf16_fixup<EPI_QKV, C>), fgrid, fblock, 0, s, p, tm); break;
        case EPI_SWIGLU: hipLaunchKernelGGL((gemm_bf16_fixup<EPI_SWIGLU, C>), fgrid, fblock, 0, s, p, tm); break;
        default: break;
      }
    }
  }
  return hipGetLastError();
}

}  // namespace

int gemm_bf16_splits(int M, int N, int K) {
  return partial_half(M, N, K) ? splits_for<GemmCfgH>(M, N, K, nullptr) : splits_for<GemmCfg>(M, N, K, nullptr);
}

size_t gemm_bf16_sk_ws_bytes() {
  // the 256 x 256 tile's pieces are the larger
  return (size_t)kMaxSkGroups * 2 * GemmCfg::WAVES * 64 * GemmCfg::ACC4 * 4 * sizeof(float);
}

hipError_t launch_gemm_bf16(GemmEpi epi, const GemmParams& p, hipStream_t s) {
  bool half;
  if (epi == EPI_PARTIAL) {
    half = partial_half(p.M, p.N, p.K);
  } else {
    half = plan_cfg<GemmCfgH>(epi, p).cost < plan_cfg<GemmCfg>(epi, p).cost;
  }
  return half ? launch_plan<GemmCfgH>(epi, p, plan_cfg<GemmCfgH>(epi, p), s)
              : launch_plan<GemmCfg>(epi, p, plan_cfg<GemmCfg>(epi, p), s);
}

}  // namespace acache
