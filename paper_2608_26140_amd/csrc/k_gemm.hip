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
// Workgroup tile: 256 weight rows x 256 activation rows x 64 K, 8 waves
// (2 along N x 4 along M, two per SIMD), each wave 128 x 64 = 4 x 2 MFMA
// 32x32x16 tiles.  LDS is double buffered with one barrier per K step;
// global loads for step k+1 are in flight while step k computes.  Rows are
// padded to 144 bytes so the 16-lane groups of a ds_read_b128 hit distinct
// banks.  Workgroups are renumbered so that each XCD (8 per chip, own L2)
// receives a contiguous run of tiles with the M index fastest: the tiles
// sharing one weight tile run on the same L2.
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
  int sk_first;    // first logical tile of the stream-K region
  int sk_units;    // K steps in the stream-K region
  int sk_groups;   // workgroups sharing the stream-K region (0: none)
  float* sk_part;  // [sk_groups][2][THREADS * ACC4 * 4] partial accumulators
};

constexpr int kGroupM = 8;       // M tiles per raster group
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
                                         int sp, int wn, int wm, int lane, const double* inv_freq) {
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
            v[j] = gt / (1.f + __expf(-gt)) * up;
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
        const double ang_pos = (double)p.pos[m];
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            float lo[4], hi[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const int r = 4 * g + j;
              const int d = a * 32 + 8 * g + 4 * hl + j;
              float sn, cs;
              rotary_sincos(ang_pos * inv_freq[d], &sn, &cs);
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

__device__ __forceinline__ void init_inv_freq(double* inv_freq, const GemmParams& p, int tid) {
  if (tid < 64) inv_freq[tid] = exp2(-(2.0 * tid / 128.0) * log2((double)p.rope_base));
}

template <int EPI, class C>
__global__ __launch_bounds__(C::THREADS) void gemm_bf16_kernel(GemmParams p, TileMap tm) {
  constexpr int BN = C::BN, BM = C::BM, BK = C::BK, LDK = C::LDK, FM = C::FM;
  __shared__ __attribute__((aligned(16))) bf16 sW[2][BN * LDK];
  __shared__ __attribute__((aligned(16))) bf16 sX[2][BM * LDK];
  __shared__ double inv_freq[64];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wn = wave % C::WN, wm = wave / C::WN;
  const int F = p.N >> 1;
  const bf16* __restrict__ X = (const bf16*)p.X;
  const bf16* __restrict__ W = (const bf16*)p.W;
  const int K = p.K;
  const int nk_tile = tm.nk;
  const int w = logical_block();
  if constexpr (EPI == EPI_QKV) init_inv_freq(inv_freq, p, tid);

  const int arow = wn * 128 + (lane & 31);
  const int brow = wm * C::WAVE_M + (lane & 31);
  const int kofs = (lane >> 5) * 8;
  constexpr int KS = BK / 16;
  constexpr int NCH = C::W_CHUNKS + C::X_CHUNKS;

  f32x16 acc[4][FM];
  // Work items: dp_rounds whole tiles, then this workgroup's stream-K range.
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
      kb = -1;  // from the split index
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
    const int k0 = kb * BK;
    const int nk = kn;

    // global -> register staging, 16 B chunks; 32-bit element offsets from
    // uniform base pointers keep the address registers few
    int woff[C::W_CHUNKS], xoff[C::X_CHUNKS];
    int wdst[C::W_CHUNKS], xdst[C::X_CHUNKS];
#pragma unroll
    for (int i = 0; i < C::W_CHUNKS; ++i) {
      const int q = tid + i * C::THREADS;
      const int r = q / C::CPR, ch = q % C::CPR;
      woff[i] = weight_row<EPI, BN>(nt, r, F) * K + k0 + ch * 8;
      wdst[i] = r * LDK + ch * 8;
    }
#pragma unroll
    for (int i = 0; i < C::X_CHUNKS; ++i) {
      const int q = tid + i * C::THREADS;
      const int r = q / C::CPR, ch = q % C::CPR;
      const int m = min(mt * BM + r, p.M - 1);
      xoff[i] = m * K + k0 + ch * 8;
      xdst[i] = r * LDK + ch * 8;
    }
    // loads of K step kt+1 are issued at the start of step kt and stored to
    // the other LDS buffer before its barrier
    u32x4 stage[NCH];
    auto load_global = [&](int kt) {
      const int ko = kt * BK;
#pragma unroll
      for (int i = 0; i < C::W_CHUNKS; ++i) stage[i] = *reinterpret_cast<const u32x4*>(W + woff[i] + ko);
#pragma unroll
      for (int i = 0; i < C::X_CHUNKS; ++i)
        stage[C::W_CHUNKS + i] = *reinterpret_cast<const u32x4*>(X + xoff[i] + ko);
    };
    auto store_lds = [&](int buf) {
#pragma unroll
      for (int i = 0; i < C::W_CHUNKS; ++i) *reinterpret_cast<u32x4*>(&sW[buf][wdst[i]]) = stage[i];
#pragma unroll
      for (int i = 0; i < C::X_CHUNKS; ++i)
        *reinterpret_cast<u32x4*>(&sX[buf][xdst[i]]) = stage[C::W_CHUNKS + i];
    };

#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < FM; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;

    // MFMA fragments are double buffered in registers: the reads of k slice
    // s+1 are issued before the MFMAs of slice s, so LDS latency overlaps
    // with matrix work instead of stalling the wave.
    bf16x8 af[2][4], bfr[2][FM];
    auto read_frags = [&](const bf16* w_s, const bf16* x_s, int s, int slot) {
#pragma unroll
      for (int a = 0; a < 4; ++a)
        af[slot][a] = *reinterpret_cast<const bf16x8*>(w_s + (arow + a * 32) * LDK + s * 16 + kofs);
#pragma unroll
      for (int b = 0; b < FM; ++b)
        bfr[slot][b] = *reinterpret_cast<const bf16x8*>(x_s + (brow + b * 32) * LDK + s * 16 + kofs);
    };
    auto mfma_step = [&](int slot) {
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < FM; ++b) acc[a][b] = mfma32x32x16(af[slot][a], bfr[slot][b], acc[a][b]);
    };
    // K step kt (LDS buffer kt&1): its first fragments are already in
    // registers.  The MFMAs of its last 16-wide slice are issued after the
    // barrier, behind the fragment reads of the next K step, so the wait for
    // those reads overlaps matrix work.
    auto step = [&](int kt, int par) {
      const bf16* w_s = sW[par];
      const bf16* x_s = sX[par];
      const bool more = kt + 1 < nk;
      if (more) load_global(kt + 1);
#pragma unroll
      for (int s = 0; s + 1 < KS; ++s) {
        read_frags(w_s, x_s, s + 1, (s + 1) & 1);
        __builtin_amdgcn_sched_barrier(0);
        mfma_step(s & 1);
        __builtin_amdgcn_sched_barrier(0);
      }
      if (more) store_lds(par ^ 1);
      __syncthreads();
      if (more) read_frags(sW[par ^ 1], sX[par ^ 1], 0, KS & 1);
      __builtin_amdgcn_sched_barrier(0);
      mfma_step((KS - 1) & 1);
      __builtin_amdgcn_sched_barrier(0);
    };

    // every wave has finished reading LDS for the previous item
    __syncthreads();
    load_global(0);
    store_lds(0);
    __syncthreads();
    read_frags(sW[0], sX[0], 0, 0);
    int kt = 0;
    for (; kt + 1 < nk; kt += 2) {
      step(kt, 0);
      step(kt + 1, 1);
    }
    if (kt < nk) step(kt, 0);

    if (sk && kn < nk_tile) {
      float* slot = tm.sk_part + ((size_t)(w * 2 + piece) * C::WAVES + wave) * (64 * C::ACC4 * 4);
      store_partial<C>(slot, acc, lane);
      ++piece;
    } else {
      if (sk) ++piece;
      epilogue<EPI, C>(p, acc, nt, mt, sp, wn, wm, lane, inv_freq);
    }
  }
}

// Stream-K fixup: block = one wave of one split tile of the stream-K region.
// Sums the tile's pieces in workgroup order and runs the epilogue.
template <int EPI, class C>
__global__ __launch_bounds__(64) void gemm_bf16_fixup(GemmParams p, TileMap tm) {
  __shared__ double inv_freq[64];
  const int lane = threadIdx.x;
  const int s = blockIdx.x / C::WAVES, wave = blockIdx.x % C::WAVES;
  const int wn = wave % C::WN, wm = wave / C::WN;
  const int nk_tile = tm.nk;
  const int first = sk_owner(tm, s * nk_tile), last = sk_owner(tm, (s + 1) * nk_tile - 1);
  if (first == last) return;  // the tile was finished by one workgroup
  if constexpr (EPI == EPI_QKV) {
    init_inv_freq(inv_freq, p, lane);
    __syncthreads();
  }
  f32x16 acc[4][C::FM];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < C::FM; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;
  for (int w = first; w <= last; ++w) {
    // piece 0 of w if w's range starts in this tile, else its piece 1
    const int piece = sk_start(tm, w) / nk_tile == s ? 0 : 1;
    add_partial<C>(tm.sk_part + ((size_t)(w * 2 + piece) * C::WAVES + wave) * (64 * C::ACC4 * 4), acc, lane);
  }
  int nt, mt, sp;
  tile_coords(tm, tm.sk_first + s, nt, mt, sp);
  epilogue<EPI, C>(p, acc, nt, mt, sp, wn, wm, lane, inv_freq);
}

}  // namespace

// 8 waves (2 per SIMD) on a 256 x 256 tile, each wave 128 x 64; BK 64.
using GemmCfg = Cfg<256, 256, 2, 4, 64>;

namespace {

int cu_count() {
  static std::atomic<int> cached[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return kMaxSkGroups;
  int n = cached[dev].load(std::memory_order_relaxed);
  if (n <= 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = kMaxSkGroups;
    cached[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

// K splits for the split-K partial epilogue.  Cost in K steps of one
// workgroup, on kMaxSkGroups CUs (fixed, so the workspace plan and the
// launch agree on any device): ceil(T s / G) rounds of ceil(nk / s) steps,
// plus s fp32 slices of M x N written here and read back by the reduction,
// about M N 8 / 9.5e6 K steps each at HBM speed.  Splits need not divide
// nk; each keeps at least kMinSkSteps steps.
template <class C>
int splits_for(int M, int N, int K) {
  const int tiles = ((M + C::BM - 1) / C::BM) * (N / C::BN);
  const int nk = K / C::BK;
  const int G = kMaxSkGroups;
  const double slice = (double)M * N * 8.0 / 9.5e6;
  int best = 1;
  double best_cost = 1e30;
  for (int s = 1; s <= kMaxSplits && nk / s >= kMinSkSteps; ++s) {
    const double cost = (double)((tiles * s + G - 1) / G) * ((nk + s - 1) / s) + s * slice;
    if (cost < best_cost) {
      best_cost = cost;
      best = s;
    }
  }
  return best;
}

template <class C>
hipError_t launch_cfg(GemmEpi epi, const GemmParams& p, hipStream_t s) {
  TileMap tm = {};
  tm.m_tiles = (p.M + C::BM - 1) / C::BM;
  tm.n_tiles = epi == EPI_SWIGLU ? (p.N / 2) / (C::BN / 2) : p.N / C::BN;
  tm.splits = epi == EPI_PARTIAL ? p.splits : 1;
  tm.nk = p.K / C::BK;
  const int tiles = tm.m_tiles * tm.n_tiles * tm.splits;
  const int nk = tm.nk;
  int grid = tiles;
  tm.dp_rounds = 1;
  tm.dp_stride = tiles;
  int sk_tiles = 0;
  if (epi != EPI_PARTIAL && p.sk_ws && nk >= kMinSkSteps) {
    // Cost in K steps of one workgroup.  Data-parallel: ceil(T / G) whole
    // tiles.  Stream-K with g workgroups on the e tiles left after r full
    // rounds: r whole tiles, ceil(e nk / g) steps, and the partial pieces
    // (at most e + g, each 256 KB written and read back once), which cost
    // about 1/16 of a K step each at HBM speed.  With g >= e every range
    // spans at most nk steps and so touches at most two tiles (the two
    // partial slots of a workgroup).
    const int G = std::min(cu_count(), kMaxSkGroups);
    const int r = tiles / G, e = tiles % G;
    const double dp_cost = (double)((tiles + G - 1) / G) * nk;
    double best = dp_cost;
    int best_g = 0;
    for (int g = e; e > 0 && g <= G; ++g) {
      const double cost = (double)r * nk + (double)((e * nk + g - 1) / g) + (e + g) / 16.0;
      if (cost < best) {
        best = cost;
        best_g = g;
      }
    }
    if (best_g > 0) {
      tm.dp_rounds = r;
      tm.dp_stride = G;
      tm.sk_first = r * G;
      tm.sk_units = e * nk;
      tm.sk_groups = best_g;
      tm.sk_part = p.sk_ws;
      grid = r > 0 ? G : best_g;
      sk_tiles = e;
    }
  }
  const dim3 block(C::THREADS);
  switch (epi) {
    case EPI_STORE: hipLaunchKernelGGL((gemm_bf16_kernel<EPI_STORE, C>), dim3(grid), block, 0, s, p, tm); break;
    case EPI_ACCUM: hipLaunchKernelGGL((gemm_bf16_kernel<EPI_ACCUM, C>), dim3(grid), block, 0, s, p, tm); break;
    case EPI_PARTIAL: hipLaunchKernelGGL((gemm_bf16_kernel<EPI_PARTIAL, C>), dim3(grid), block, 0, s, p, tm); break;
    case EPI_QKV: hipLaunchKernelGGL((gemm_bf16_kernel<EPI_QKV, C>), dim3(grid), block, 0, s, p, tm); break;
    case EPI_SWIGLU: hipLaunchKernelGGL((gemm_bf16_kernel<EPI_SWIGLU, C>), dim3(grid), block, 0, s, p, tm); break;
  }
  if (sk_tiles > 0) {
    const dim3 fgrid(sk_tiles * C::WAVES), fblock(64);
    switch (epi) {
      case EPI_STORE: hipLaunchKernelGGL((gemm_bf16_fixup<EPI_STORE, C>), fgrid, fblock, 0, s, p, tm); break;
      case EPI_ACCUM: hipLaunchKernelGGL((gemm_bf16_fixup<EPI_ACCUM, C>), fgrid, fblock, 0, s, p, tm); break;
      case EPI_QKV: hipLaunchKernelGGL((gemm_bf16_fixup<EPI_QKV, C>), fgrid, fblock, 0, s, p, tm); break;
      case EPI_SWIGLU: hipLaunchKernelGGL((gemm_bf16_fixup<EPI_SWIGLU, C>), fgrid, fblock, 0, s, p, tm); break;
      default: break;
    }
  }
  return hipGetLastError();
}

}  // namespace

int gemm_bf16_splits(int M, int N, int K) { return splits_for<GemmCfg>(M, N, K); }

size_t gemm_bf16_sk_ws_bytes() {
  return (size_t)kMaxSkGroups * 2 * GemmCfg::WAVES * 64 * GemmCfg::ACC4 * 4 * sizeof(float);
}

hipError_t launch_gemm_bf16(GemmEpi epi, const GemmParams& p, hipStream_t s) {
  return launch_cfg<GemmCfg>(epi, p, s);
}

}  // namespace acache
