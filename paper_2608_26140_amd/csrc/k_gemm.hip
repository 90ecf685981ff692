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
// Workgroup tile: 256 weight rows x 128 activation rows x 64 K, 4 waves
// (2 x 2), each wave 128 x 64 = 4 x 2 MFMA 32x32x16 tiles.  LDS is double
// buffered with one barrier per K step; global loads for step k+1 are in
// flight while step k computes.  Rows are padded to 144 bytes so the
// 16-lane groups of a ds_read_b128 hit distinct banks.  Workgroups are
// renumbered so that each XCD (8 per chip, own L2) receives a contiguous run
// of tiles with the M index fastest: the tiles sharing one weight tile run on
// the same L2.
//
// Epilogues: plain store, accumulate, fp32 split-K partials, Q/K/V with
// rotary embedding and the K/V store to pool slots, and SwiGLU.
#include <cstdlib>

#include "device.h"
#include "internal.h"

namespace acache {

namespace {

// Tile configurations.  Every wave covers 128 weight rows (one attention
// head, or 64 gate + 64 up rows) and WAVE_M activation rows.
template <int BN_, int BM_, int WN_, int WM_, int BK_, int STAGES_ = 2>
struct Cfg {
  static constexpr int STAGES = STAGES_;  // register stages of global prefetch
  static constexpr int BN = BN_;       // weight rows per workgroup
  static constexpr int BM = BM_;       // activation rows per workgroup
  static constexpr int WN = WN_;       // waves along N
  static constexpr int WM = WM_;       // waves along M
  static constexpr int BK = BK_;       // K per LDS stage
  static constexpr int LDK = BK + 8;   // padded LDS row (elements)
  static constexpr int THREADS = 64 * WN * WM;
  static constexpr int WAVE_M = BM / WM;
  static constexpr int FM = WAVE_M / 32;  // activation fragments per wave
  static constexpr int CPR = BK / 8;      // 16-byte chunks per row
  static constexpr int W_CHUNKS = BN * CPR / THREADS;
  static constexpr int X_CHUNKS = BM * CPR / THREADS;
  static_assert(BN / WN == 128, "a wave spans 128 weight rows");
  static_assert(WAVE_M % 32 == 0 && FM >= 1, "wave M extent");
  static_assert(BK % 32 == 0, "an even number of 16-wide K slices per stage");
  static_assert(BN * CPR % THREADS == 0 && BM * CPR % THREADS == 0, "load split");
};

typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4;

struct TileMap {
  int n_tiles, m_tiles, splits, k_per_split;
};

constexpr int kGroupM = 8;  // M tiles per raster group

// Workgroup -> (n tile, m tile, split).  Workgroups are dealt round-robin to
// the 8 XCDs, so renumber them to give each XCD a contiguous range of
// logical tiles; inside a split, tiles run in groups of kGroupM M tiles with
// the M index fastest, so the workgroups resident at one time on an XCD
// share both their weight tiles and their activation tiles in its L2.
__device__ __forceinline__ void tile_of(const TileMap& tm, int& nt, int& mt, int& sp) {
  const int nb = gridDim.x;
  const int i = blockIdx.x;
  const int q = nb >> 3, r = nb & 7;
  const int x = i & 7, slot = i >> 3;
  const int t = x * q + min(x, r) + slot;
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

template <int EPI, class C>
__global__ __launch_bounds__(C::THREADS) void gemm_bf16_kernel(GemmParams p, TileMap tm) {
  constexpr int BN = C::BN, BM = C::BM, BK = C::BK, LDK = C::LDK, FM = C::FM;
  __shared__ __attribute__((aligned(16))) bf16 sW[2][BN * LDK];
  __shared__ __attribute__((aligned(16))) bf16 sX[2][BM * LDK];
  __shared__ double inv_freq[64];

  int nt, mt, sp;
  tile_of(tm, nt, mt, sp);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wn = wave % C::WN, wm = wave / C::WN;
  const int F = p.N >> 1;
  const bf16* __restrict__ X = (const bf16*)p.X;
  const bf16* __restrict__ W = (const bf16*)p.W;
  const int K = p.K;
  const int k0 = sp * tm.k_per_split;
  const int nk = tm.k_per_split / BK;

  if constexpr (EPI == EPI_QKV) {
    if (tid < 64) inv_freq[tid] = exp2(-(2.0 * tid / 128.0) * log2((double)p.rope_base));
  }

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
  // With two register stages the global loads of K step kt+2 are issued
  // while step kt computes, and the stores of step kt+1 into LDS are spread
  // over step kt's MFMA slices; with one stage, loads of step kt+1 are issued
  // at the start of step kt and stored before its barrier.
  constexpr int NCH = C::W_CHUNKS + C::X_CHUNKS;
  u32x4 stage[C::STAGES][NCH];
  auto load_global = [&](int kt, int st) {
    const int ko = kt * BK;
#pragma unroll
    for (int i = 0; i < C::W_CHUNKS; ++i) stage[st][i] = *reinterpret_cast<const u32x4*>(W + woff[i] + ko);
#pragma unroll
    for (int i = 0; i < C::X_CHUNKS; ++i)
      stage[st][C::W_CHUNKS + i] = *reinterpret_cast<const u32x4*>(X + xoff[i] + ko);
  };
  auto store_chunk = [&](int buf, int st, int i) {
    if (i < C::W_CHUNKS)
      *reinterpret_cast<u32x4*>(&sW[buf][wdst[i]]) = stage[st][i];
    else
      *reinterpret_cast<u32x4*>(&sX[buf][xdst[i - C::W_CHUNKS]]) = stage[st][i];
  };
  auto store_lds = [&](int buf, int st) {
#pragma unroll
    for (int i = 0; i < NCH; ++i) store_chunk(buf, st, i);
  };

  f32x16 acc[4][FM];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < FM; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;

  const int arow = wn * 128 + (lane & 31);
  const int brow = wm * C::WAVE_M + (lane & 31);
  const int kofs = (lane >> 5) * 8;

  // MFMA fragments are double buffered in registers: the reads of k step
  // s+1 are issued before the MFMAs of step s, so LDS latency overlaps with
  // matrix work instead of stalling the wave.
  constexpr int KS = BK / 16;
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
    if constexpr (C::STAGES == 2) {
      if (kt + 2 < nk) load_global(kt + 2, par);
    } else {
      if (more) load_global(kt + 1, 0);
    }
#pragma unroll
    for (int s = 0; s + 1 < KS; ++s) {
      read_frags(w_s, x_s, s + 1, (s + 1) & 1);
      if constexpr (C::STAGES == 2) {
        if (more) {
#pragma unroll
          for (int i = s * NCH / (KS - 1); i < (s + 1) * NCH / (KS - 1); ++i) store_chunk(par ^ 1, par ^ 1, i);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
      mfma_step(s & 1);
      __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (C::STAGES == 1) {
      if (more) store_lds(par ^ 1, 0);
    }
    __syncthreads();
    if (more) read_frags(sW[par ^ 1], sX[par ^ 1], 0, KS & 1);
    __builtin_amdgcn_sched_barrier(0);
    mfma_step((KS - 1) & 1);
    __builtin_amdgcn_sched_barrier(0);
  };

  load_global(0, 0);
  store_lds(0, 0);
  if (C::STAGES == 2 && nk > 1) load_global(1, C::STAGES - 1);
  __syncthreads();
  read_frags(sW[0], sX[0], 0, 0);
  int kt = 0;
  for (; kt + 1 < nk; kt += 2) {
    step(kt, 0);
    step(kt + 1, 1);
  }
  if (kt < nk) step(kt, 0);

  // ------------------------------------------------------------ epilogue
  // acc[a][b][r] = C[m = mbase + 32b + lane%32][n = nbase + 32a + 8(r/4) + 4(lane/32) + r%4]
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
      float out[4][16];
      if (!is_v) {
        const double ang_pos = (double)p.pos[m];
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int d = a * 32 + 8 * (r >> 2) + 4 * hl + (r & 3);
            double ang = ang_pos * inv_freq[d];
            ang -= 6.283185307179586 * rint(ang * 0.15915494309189535);
            float sn, cs;
            sincosf((float)ang, &sn, &cs);
            const float x1 = acc[a][b][r], x2 = acc[a + 2][b][r];
            out[a][r] = x1 * cs - x2 * sn;
            out[a + 2][r] = x2 * cs + x1 * sn;
          }
      } else {
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
          for (int r = 0; r < 16; ++r) out[a][r] = acc[a][b][r];
      }
      bf16* dst;
      if (col0 < p.hq_cols) {
        dst = (bf16*)p.q_out + (int64_t)m * p.hq_cols + col0;
      } else {
        const int64_t slot = p.write_slots[m];
        if (slot < 0 || slot >= p.n_slots) continue;
        const int c = is_v ? col0 - p.hq_cols - p.hkv_cols : col0 - p.hq_cols;
        dst = (bf16*)(is_v ? p.v_pool : p.k_pool) + slot * p.pool_ld + c;
      }
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const float v[4] = {out[a][4 * g], out[a][4 * g + 1], out[a][4 * g + 2], out[a][4 * g + 3]};
          store4(dst + a * 32 + g * 8 + hl * 4, v);
        }
    }
  }
}

}  // namespace

// 8 waves (2 per SIMD) on a 256 x 256 tile, each wave 128 x 64; BK 64 with one
// register stage: measured fastest on every projection shape of the workloads.
using GemmCfg = Cfg<256, 256, 2, 4, 64, 1>;

template <class C>
int splits_for(int M, int N, int K) {
  const int tiles = ((M + C::BM - 1) / C::BM) * (N / C::BN);
  const int ksteps = K / C::BK;
  int best = 1;
  // enough workgroups to cover 256 CUs about twice, K per split >= 512
  for (int s = 1; s <= 8; ++s) {
    if (ksteps % s || (K / s) < 512) continue;
    best = s;
    if (tiles * s >= 448) break;
  }
  return best;
}

int gemm_bf16_splits(int M, int N, int K) { return splits_for<GemmCfg>(M, N, K); }

template <class C>
hipError_t launch_cfg(GemmEpi epi, const GemmParams& p, hipStream_t s) {
  TileMap tm;
  tm.m_tiles = (p.M + C::BM - 1) / C::BM;
  tm.n_tiles = epi == EPI_SWIGLU ? (p.N / 2) / (C::BN / 2) : p.N / C::BN;
  tm.splits = epi == EPI_PARTIAL ? p.splits : 1;
  tm.k_per_split = p.K / tm.splits;
  const dim3 grid(tm.m_tiles * tm.n_tiles * tm.splits);
  const dim3 block(C::THREADS);
  switch (epi) {
    case EPI_STORE: hipLaunchKernelGGL((gemm_bf16_kernel<EPI_STORE, C>), grid, block, 0, s, p, tm); break;
    case EPI_ACCUM: hipLaunchKernelGGL((gemm_bf16_kernel<EPI_ACCUM, C>), grid, block, 0, s, p, tm); break;
    case EPI_PARTIAL: hipLaunchKernelGGL((gemm_bf16_kernel<EPI_PARTIAL, C>), grid, block, 0, s, p, tm); break;
    case EPI_QKV: hipLaunchKernelGGL((gemm_bf16_kernel<EPI_QKV, C>), grid, block, 0, s, p, tm); break;
    case EPI_SWIGLU: hipLaunchKernelGGL((gemm_bf16_kernel<EPI_SWIGLU, C>), grid, block, 0, s, p, tm); break;
  }
  return hipGetLastError();
}

hipError_t launch_gemm_bf16(GemmEpi epi, const GemmParams& p, hipStream_t s) {
  return launch_cfg<GemmCfg>(epi, p, s);
}

}  // namespace acache
