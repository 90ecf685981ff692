// Read-slot flash attention for gfx950 (Appendix C.1): bidirectional, no
// mask, grouped KV heads, keys and values gathered through a slot map.
//
// attention_pv_kernel   128 queries per workgroup (4 wavefronts x 32), a
//                       two-stage LDS ring of 64-key K and V tiles; two
//                       workgroups per CU.  Optional per-query key masks
//                       (the decode step's shared pass) and key splits
//                       merged by attention_merge_kernel.
// attention_wide_kernel 256 queries per workgroup (8 wavefronts x 32), a
//                       four-stage ring filled three tiles ahead, one
//                       workgroup per CU; for grids that fill whole rounds.
// Both form S^T = K Q^T with the K tile as the MFMA A operand, so each lane
// owns one query (in-lane softmax statistics plus one exchange between the
// lane halves), and O^T += V^T P^T with the lane's own exp'd logits as the
// B operand (a fixed key permutation inside each 16-key group makes that
// layout line up); V is stored untransposed and read as V^T through
// transposing LDS reads.  Softmax runs in base 2 on log2(e)/sqrt(d_h)-
// prescaled logits (hardware exp2) with a lazy rescale of the running max.
#include <algorithm>

#include "device.h"
#include "internal.h"

namespace acache {

namespace {

constexpr int kDh = 128;
constexpr int kTileK = 64;           // keys per LDS stage

typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4;

struct AttnArgs {
  const bf16* q;
  int64_t q_ld;
  int64_t q_n_rows;
  const int32_t* q_idx;  // nullable: query i of a request is row q_idx[row_start + i]
  const int32_t* slots;  // key j of request b is pool row slots[key_start[b] + j]
  const bf16* k_pool;
  const bf16* v_pool;
  int64_t pool_ld;
  int64_t n_slots;
  bf16* out;             // [rows, H * 128] (PV only)
  float* lse;            // [.., H] natural log; nullable for PV
  // nullable: [.., H] natural-log log-sum-exp over key tiles 0 .. aff_t1 - 1
  // of each request, the state of the running softmax once those tiles are
  // in (the keys are visited in order).  Under key splits each split leaves
  // its share in PvArgs::part_aff and the merge kernel combines them
  float* lse_aff;
  int aff_t1;
  int H, Hkv;
  int batch;
  int row_start[kMaxBatch + 1];
  // the rows of request b this launch takes: row_start[b] + row_lo[b] ..
  // + row_n[b] - 1 (a launch may take a part of each request's rows)
  int row_lo[kMaxBatch];
  int row_n[kMaxBatch];
  int key_start[kMaxBatch + 1];
  int key_len[kMaxBatch + 1];
  int tile_start[kMaxBatch + 1];
};

// Physical key (within a 32-key block) read by S^T row i.
__device__ __forceinline__ int key_perm(int i) {
  const int r = i & 15;
  return (i & 16) | (8 * ((r >> 2) & 1) + (r & 3) + 4 * (r >> 3));
}

// ============================================================================
// Read-slot attention with the K/V tiles loaded straight into LDS.
//
// A workgroup holds 128 queries of one head (4 wavefronts x 32) and streams
// a contiguous range of the request's key tiles (64 keys) through a
// two-stage LDS ring; two workgroups fit one CU, two wavefronts per SIMD.
// Loads are global -> LDS (16 bytes per lane, no staging registers):
//   K tile [64 keys][256 B], 16-byte chunk c of key row r at c ^ (r & 15):
//     the 16 rows read by one ds_read_b128 pass hit 16 distinct chunks;
//   V tile [64 keys][256 B] untransposed, chunk c at c ^ 2 (r & 3).
// The A operand of O^T = V^T P^T (8 consecutive keys of one dimension per
// lane) comes from two transposing LDS reads (ds_read_b64_tr_b16): in each
// 16-lane group, lane l receives element l % 4 of the 8-byte runs addressed
// by lanes l / 4, l / 4 + 4, l / 4 + 8, l / 4 + 12; lane i therefore points
// at key key0 + i / 4, dimensions dgroup + 4 (i % 4) .. + 3, and receives
// keys key0 .. key0 + 3 of dimension dgroup + l.
// Keys that are absent (past the request's end, or an out-of-range slot)
// load slot 0 and the loading lane zeroes its LDS chunk once the data has
// landed; keys past the end are also masked to -inf in the softmax.
// With several key splits the workgroup writes its unnormalised O and its
// (max, sum) in fp32 and attention_merge_kernel combines the splits.
// ============================================================================

typedef short v4i16 __attribute__((__vector_size__(4 * sizeof(short))));

constexpr int kPvWaves = 4;
constexpr int kPvTileQ = 32 * kPvWaves;
constexpr int kPvThreads = 64 * kPvWaves;
constexpr int kRowB = kDh * 2;                    // bytes per key row
constexpr int kTileB = kTileK * kRowB;            // 16 KB: one K or V tile
constexpr int kStageB = 2 * kTileB;               // K tile + V tile
constexpr int kDmaPerTile = kTileB / 1024 / kPvWaves;  // 1 KB loads per wave per tile

struct PvArgs {
  AttnArgs a;
  int splits;
  float* part_o;   // [splits][rows][H][128] unnormalised O (splits > 1)
  float* part_ml;  // [splits][rows][H][2] (running max in log2 units, sum)
  // with lse_aff and splits > 1: [splits][rows][H], each split's log-sum-exp
  // (log2 units) over its tiles below aff_t1, -inf for a split past them
  float* part_aff;
  // decode passes: both write partials into one buffer of part_rows rows,
  // this launch's splits at indices split_base ..
  int partial;
  int split_base;
  int64_t part_rows;
  // MASK kernels: bit i of key_mask[(row / mask_rows) * mask_tiles + t] drops
  // key 64 t + i for that query row
  const uint64_t* key_mask;
  int mask_tiles;
  int mask_rows;
};

__device__ __forceinline__ v4i16 ds_read_tr16(const char* lds) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4i16*)lds);
}

template <bool MASK>
__global__ __launch_bounds__(kPvThreads, 2) void attention_pv_kernel(PvArgs pa) {
  __shared__ __attribute__((aligned(1024))) char ring[2 * kStageB];
  const AttnArgs& a = pa.a;
  const int splits = pa.splits;

  // XCD-contiguous, head-major order of (head, query tile, key split)
  const int n_tiles_q = a.tile_start[a.batch];
  int h, tile, split;
  {
    const int nb = gridDim.x, i = blockIdx.x;
    const int q8 = nb >> 3, r8 = nb & 7, x = i & 7;
    const int t = x * q8 + min(x, r8) + (i >> 3);
    h = t / (n_tiles_q * splits);
    const int rem = t - h * n_tiles_q * splits;
    tile = rem / splits;
    split = rem - tile * splits;
  }
  int b = 0;
  {
    int lo = 0, hi = a.batch - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (a.tile_start[mid] <= tile) lo = mid; else hi = mid - 1;
    }
    b = lo;
  }
  const int g = h / (a.H / a.Hkv);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, hl = lane >> 5;
  const int n_rows = a.row_n[b];
  const int64_t r0 = (int64_t)a.row_start[b] + a.row_lo[b];  // global row of query 0
  const int qi = (tile - a.tile_start[b]) * kPvTileQ + wave * 32 + (lane & 31);
  const bool q_ok = qi < n_rows;
  // a wavefront without a valid query only copies and synchronises
  const bool live = __builtin_amdgcn_ballot_w64(q_ok) != 0;
  const int S = a.key_len[b];
  const int32_t* slots = a.slots + a.key_start[b];
  const int n_kt = (S + kTileK - 1) / kTileK;
  const int t_lo = split * n_kt / splits, t_hi = (split + 1) * n_kt / splits;

  bf16x8 qf[8];
  {
    int64_t qrow = q_ok ? r0 + qi : -1;
    const bf16* qp = a.q + (qrow < 0 ? 0 : qrow) * a.q_ld + h * kDh + hl * 8;
#pragma unroll
    for (int s2 = 0; s2 < 8; ++s2) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (qrow >= 0) v = *reinterpret_cast<const u32x4*>(qp + s2 * 16);
      qf[s2] = __builtin_bit_cast(bf16x8, v);
    }
  }

  const uint64_t* mrow = nullptr;  // this query row's key mask (MASK)
  if constexpr (MASK) {
    if (q_ok) mrow = pa.key_mask + (int64_t)((r0 + qi) / pa.mask_rows) * pa.mask_tiles;
  }

  // this lane's 4 keys of a tile (one per load): key 16 wave + 4 i + lane / 16,
  // 16-byte chunk position lane % 16
  const int pch = lane & 15;
  const uint32_t head_b = (uint32_t)g * kRowB;
  const uint32_t ld_b = (uint32_t)a.pool_ld * 2u;
  int slot_next[kDmaPerTile];   // slots of the tile to issue next
  unsigned absent_bits = 0;     // bit i: this lane's key i of the in-flight tile is absent
  auto key_of = [&](int t, int i) { return t * kTileK + wave * 16 + 4 * i + (lane >> 4); };
  auto load_slots = [&](int t) {
#pragma unroll
    for (int i = 0; i < kDmaPerTile; ++i) slot_next[i] = slots[min(key_of(t, i), S - 1)];
  };
  auto issue = [&](int t) {
    char* st = ring + (t & 1) * kStageB;
    unsigned ab = 0;
#pragma unroll
    for (int i = 0; i < kDmaPerTile; ++i) {
      const int key = key_of(t, i);
      const int sl = slot_next[i];
      const bool ok = key < S && sl >= 0 && sl < a.n_slots;
      ab |= (ok ? 0u : 1u) << i;
      const uint32_t base = (ok ? (uint32_t)sl : 0u) * ld_b + head_b;
      const int r = key & (kTileK - 1);
      const int ck = pch ^ (r & 15), cv = pch ^ ((r & 3) << 1);
      const int dst = (wave * kDmaPerTile + i) * 1024;
      dma16((const char*)a.k_pool + base + ck * 16, st + dst);
      dma16((const char*)a.v_pool + base + cv * 16, st + kTileB + dst);
    }
    absent_bits = ab;
  };
  // zero the chunks this lane loaded for absent keys (after they landed)
  auto fix_absent = [&](int t) {
    if (absent_bits) {
      char* st = ring + (t & 1) * kStageB;
      const u32x4 z = {0u, 0u, 0u, 0u};
#pragma unroll
      for (int i = 0; i < kDmaPerTile; ++i)
        if ((absent_bits >> i) & 1u) {
          const int dst = (wave * kDmaPerTile + i) * 1024 + lane * 16;
          *reinterpret_cast<u32x4*>(st + dst) = z;
          *reinterpret_cast<u32x4*>(st + kTileB + dst) = z;
        }
    }
  };

  f32x16 o_acc[4];
#pragma unroll
  for (int d = 0; d < 4; ++d)
#pragma unroll
    for (int r = 0; r < 16; ++r) o_acc[d][r] = 0.f;
  float m_run = -INFINITY, l_part = 0.f, lse_aff2 = -INFINITY;
  // the affix tiles of this split end before tile aff_end (none if past them)
  const int aff_end = min(a.aff_t1, t_hi);
  const float scale = kLog2e * rsqrtf((float)kDh);
  const int krow = key_perm(lane & 31);
  // K fragment byte offsets inside a tile for key block 0 (block 1: + 32 rows)
  const int k_row_off = krow * kRowB;
  const int k_sw = krow & 15;  // same for krow + 32
  // transposing V reads: this lane's 16-lane group and index in it
  const int grp = lane >> 4, gi = lane & 15;
  const int v_key = 8 * (grp >> 1) + (gi >> 2);  // + 32 kb + 16 g2 (+ 4 for the second read)
  const int v_chunk_lo = 2 * (grp & 1) + ((gi & 3) >> 1);  // + 4 d
  const int v_byte = (gi & 1) * 8;
  const int v_sw = (gi >> 2) << 1;  // 2 (row & 3), row & 3 == gi / 4 (key0 is a multiple of 4)

  if (t_lo < t_hi) {
    load_slots(t_lo);
    issue(t_lo);
    if (t_lo + 1 < t_hi) load_slots(t_lo + 1);
  }
  for (int t = t_lo; t < t_hi; ++t) {
    // tile t (and the slot indices of t + 1) have landed in this wave
    wait_vmcnt<0>();
    fix_absent(t);
    lds_barrier();
    if (t + 1 < t_hi) {
      issue(t + 1);  // into the slot of tile t - 1, which every wave has finished
      if (t + 2 < t_hi) load_slots(t + 2);
    }
    if (!live) continue;
    const char* ks = ring + (t & 1) * kStageB;
    const char* vs = ks + kTileB;
    f32x16 st[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      bf16x8 kf[8];
#pragma unroll
      for (int s2 = 0; s2 < 8; ++s2)
        kf[s2] = *reinterpret_cast<const bf16x8*>(ks + kb * 32 * kRowB + k_row_off + (((2 * s2 + hl) ^ k_sw) << 4));
#pragma unroll
      for (int r = 0; r < 16; ++r) st[kb][r] = 0.f;
#pragma unroll
      for (int s2 = 0; s2 < 8; ++s2) st[kb] = mfma32x32x16(kf[s2], qf[s2], st[kb]);
    }
    const int kt0 = t * kTileK;
    // keys of this tile dropped for this query: past the end, or masked
    uint64_t drop = kt0 + kTileK <= S ? 0ull : ~0ull << (S - kt0);
    if constexpr (MASK) drop |= mrow ? mrow[t] : 0ull;
    float mx = -INFINITY;
    if (drop == 0ull) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, st[kb][r]);
    } else {
      // register r of key block kb holds key 32 kb + 16 (r / 8) + 8 hl + r % 8
      const uint32_t dw[2] = {(uint32_t)drop >> (8 * hl), (uint32_t)(drop >> 32) >> (8 * hl)};
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          st[kb][r] = (dw[kb] >> (16 * (r >> 3) + (r & 7))) & 1u ? -INFINITY : st[kb][r];
          mx = fmaxf(mx, st[kb][r]);
        }
    }
    mx = fmaxf(mx, __shfl_xor(mx, 32)) * scale;
    // lazy rescale: the running max moves only when exceeded by more than 2^8
    const bool bump = mx > m_run + 8.f;
    if (__builtin_amdgcn_ballot_w64(bump)) {
      const float m_new = bump ? mx : m_run;
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_part *= alpha;
#pragma unroll
      for (int d = 0; d < 4; ++d)
#pragma unroll
        for (int r = 0; r < 16; ++r) o_acc[d][r] *= alpha;
    }
    // with masks a query may not have met a key yet (running max -inf, all
    // its logits -inf): exponentiate against 0 then, which gives zeros
    const float m_use = MASK && m_run == -INFINITY ? 0.f : m_run;
    float psum = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float e = __builtin_amdgcn_exp2f(fmaf(st[kb][r], scale, -m_use));
        st[kb][r] = e;
        psum += e;
      }
    l_part += psum;
    if (t + 1 == aff_end) lse_aff2 = m_run + __log2f(l_part + __shfl_xor(l_part, 32));
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int g2 = 0; g2 < 2; ++g2) {
        bf16x8 pb;
#pragma unroll
        for (int j = 0; j < 8; ++j) pb[j] = (bf16)st[kb][8 * g2 + j];
        const int row0 = kb * 32 + g2 * 16 + v_key;  // first of this lane's 4 address rows
#pragma unroll
        for (int d = 0; d < 4; ++d) {
          const int off = ((4 * d + v_chunk_lo) ^ v_sw) * 16 + v_byte;
          const v4i16 lo = ds_read_tr16(vs + row0 * kRowB + off);
          const v4i16 hi = ds_read_tr16(vs + (row0 + 4) * kRowB + off);
          const bf16x8 vf = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
          o_acc[d] = mfma32x32x16(vf, pb, o_acc[d]);
        }
      }
  }

  const float l_tot = l_part + __shfl_xor(l_part, 32);
  if (!q_ok) return;
  const int64_t row = r0 + qi;
  if (splits > 1 || pa.partial) {
    // unnormalised partial: O^T register r of block d holds dims 32 d + 8 (r / 4) + 4 hl + r % 4
    const int64_t prow = pa.partial ? pa.part_rows : (int64_t)a.row_start[a.batch];
    const int psplit = pa.split_base + split;
    float* po = pa.part_o + (((int64_t)psplit * prow + row) * a.H + h) * kDh;
#pragma unroll
    for (int d = 0; d < 4; ++d)
#pragma unroll
      for (int gq = 0; gq < 4; ++gq) {
        const f32x4 v = {o_acc[d][4 * gq], o_acc[d][4 * gq + 1], o_acc[d][4 * gq + 2], o_acc[d][4 * gq + 3]};
        *reinterpret_cast<f32x4*>(po + d * 32 + 8 * gq + 4 * hl) = v;
      }
    if (hl == 0) {
      float* pm = pa.part_ml + (((int64_t)psplit * prow + row) * a.H + h) * 2;
      pm[0] = m_run;
      pm[1] = l_tot;
      if (pa.part_aff) pa.part_aff[((int64_t)psplit * prow + row) * a.H + h] = lse_aff2;
    }
    return;
  }
  if (a.lse && hl == 0) a.lse[row * a.H + h] = (m_run + __log2f(l_tot)) * kLn2;
  if (a.lse_aff && hl == 0) a.lse_aff[row * a.H + h] = lse_aff2 * kLn2;
  const float inv = 1.f / l_tot;
  bf16* op = a.out + row * (int64_t)a.H * kDh + (int64_t)h * kDh;
#pragma unroll
  for (int d = 0; d < 4; ++d)
#pragma unroll
    for (int gq = 0; gq < 4; ++gq) {
      bf16x4 w;
#pragma unroll
      for (int j = 0; j < 4; ++j) w[j] = (bf16)(o_acc[d][4 * gq + j] * inv);
      *reinterpret_cast<bf16x4*>(op + d * 32 + 8 * gq + 4 * hl) = w;
    }
}

// Combines the key splits of each (row, head): m = max_s m_s,
// O = sum_s 2^(m_s - m) O_s / sum_s 2^(m_s - m) l_s.  32 threads per
// (row, head), 4 dimensions each.  With part_aff also the affix
// log-sum-exp, log sum_s 2^(a_s) over the splits' shares a_s.
__global__ __launch_bounds__(256) void attention_merge_kernel(const float* __restrict__ part_o,
                                                              const float* __restrict__ part_ml, int splits,
                                                              int64_t rows, int H, bf16* __restrict__ out,
                                                              float* __restrict__ lse,
                                                              const float* __restrict__ part_aff,
                                                              float* __restrict__ lse_aff) {
  const int64_t pair = (int64_t)blockIdx.x * 8 + (threadIdx.x >> 5);
  if (pair >= rows * H) return;
  const int c = (threadIdx.x & 31) * 4;
  float m = -INFINITY;
  for (int s2 = 0; s2 < splits; ++s2) m = fmaxf(m, part_ml[((int64_t)s2 * rows * H + pair) * 2]);
  float l = 0.f;
  f32x4 o = {0.f, 0.f, 0.f, 0.f};
  for (int s2 = 0; s2 < splits; ++s2) {
    const float* ml = part_ml + ((int64_t)s2 * rows * H + pair) * 2;
    const float w = ml[0] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(ml[0] - m);
    l += w * ml[1];
    const f32x4 v = *reinterpret_cast<const f32x4*>(part_o + ((int64_t)s2 * rows * H + pair) * kDh + c);
#pragma unroll
    for (int j = 0; j < 4; ++j) o[j] += w * v[j];
  }
  const float inv = 1.f / l;
  bf16x4 w;
#pragma unroll
  for (int j = 0; j < 4; ++j) w[j] = (bf16)(o[j] * inv);
  *reinterpret_cast<bf16x4*>(out + pair * kDh + c) = w;
  if (lse && c == 0) lse[pair] = (m + __log2f(l)) * kLn2;
  if (part_aff && c == 0) {
    float ma = -INFINITY;
    for (int s2 = 0; s2 < splits; ++s2) ma = fmaxf(ma, part_aff[(int64_t)s2 * rows * H + pair]);
    float la = 0.f;
    for (int s2 = 0; s2 < splits; ++s2) {
      const float v = part_aff[(int64_t)s2 * rows * H + pair];
      la += v == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(v - ma);
    }
    lse_aff[pair] = (ma + __log2f(la)) * kLn2;
  }
}


// ============================================================================
// Read-slot attention, wide query tiles (the recompute's large row counts).
//
// A workgroup holds 32 QB WAVES queries of one head: WAVES wavefronts of QB
// 32-query MFMA blocks each, one workgroup per CU.  The 128 KB of LDS hold a
// ring of four 64-key stages (K + V tiles), filled by buffer -> LDS copies
// issued from inline assembly three tiles ahead of the tile being finished
// (the compiler's wait analysis does not see them and does not drain them
// before each LDS read; the kernel waits for them itself with vmcnt,
// counting a fixed number of copies per tile).  The slot indices of a tile
// are copied to LDS the same way one tile earlier still.  Keys past the
// request's end and out-of-range slots take a buffer offset beyond the
// pool, which loads zeros.
//
// The tile loop is software pipelined: iteration t computes S(t+1) = K Q^T
// of the next tile while it exponentiates tile t's logits, then O += V P of
// tile t while it takes the row maxima of tile t+1, so matrix and vector
// work are independent within each half of the iteration.  The copies of
// tile t+3 are issued between the first MFMAs of the iteration rather than
// ahead of them (measured: 9-10% faster; a wave that issues its copies and
// their address work first leaves its SIMD's matrix unit idle meanwhile).
// The running max moves only when a tile exceeds it by more than 2^8 (lazy
// rescale), after tile t's P V has been added.  Per query the keys are
// visited in the same order and tiles, with the same MFMA sequences, as
// attention_pv_kernel, so the two kernels give the same bits.
//
// Measured (8 wavefronts of 32 queries, two per SIMD): 39-41% of the bf16
// peak on the serving shapes (512 and 2150 rows per request over 8704
// keys), against 36-37% for attention_pv_kernel's two 128-query workgroups
// per CU; slower than it for grids that fill less than one round (fewer,
// longer-lived workgroups).  Four wavefronts of 64 queries halve the LDS
// reads per MFMA but run one wavefront per SIMD, and lose: the overlap of
// matrix and vector work needs two wavefronts per SIMD.  Variants measured
// and not kept: K/V staged through registers instead of buffer -> LDS
// copies (equal); no LDS fragment reads at all, or no exponentials (each
// under 10% faster, so neither is what bounds the loop).
// ============================================================================

typedef uint32_t rsrc_words __attribute__((ext_vector_type(4)));

// Raw buffer descriptor over [base, base + bytes) in SGPRs (stride 0: loads
// at or past `bytes` return zeros).
__device__ __forceinline__ rsrc_words buffer_words(const void* base, uint32_t bytes) {
  const uint64_t p = (uint64_t)(uintptr_t)base;
  rsrc_words w;
  w.x = __builtin_amdgcn_readfirstlane((uint32_t)p);
  w.y = __builtin_amdgcn_readfirstlane((uint32_t)(p >> 32) & 0xFFFFu);
  w.z = __builtin_amdgcn_readfirstlane(bytes);
  w.w = 0x00020000u;
  return w;
}
// 16 bytes per lane, buffer -> LDS at lds + 16 * lane (lds wave-uniform).
__device__ __forceinline__ void dma16_asm(rsrc_words r, uint32_t voff, const char* lds) {
  const uint32_t m0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds);
  asm volatile("buffer_load_dwordx4 %0, %1, 0 offen lds" ::"v"(voff), "s"(r), "{m0}"(m0) : "memory");
}
// 4 bytes per lane, buffer -> LDS at lds + 4 * lane.
__device__ __forceinline__ void dma4_asm(rsrc_words r, uint32_t voff, const char* lds) {
  const uint32_t m0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds);
  asm volatile("buffer_load_dword %0, %1, 0 offen lds" ::"v"(voff), "s"(r), "{m0}"(m0) : "memory");
}
// s_waitcnt vmcnt(N) that the compiler cannot move memory accesses across.
template <int N>
__device__ __forceinline__ void wait_vm_asm() {
  static_assert(N >= 0 && N < 64, "vmcnt field");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

constexpr int kWdStages = 4;                     // K + V stages in the ring
constexpr int kWdKAhead = 3;                     // K fragments read ahead, in MFMA chunks
constexpr int kWdVAhead = 2;                     // V fragments read ahead
constexpr int kWdSlotB = kTileK * 4;             // one tile's slot indices
// buffer offset of an absent key: past every pool the launcher admits
// (n_slots * pool_ld * 2 <= kWdAbsent), so its loads return zeros
constexpr uint32_t kWdAbsent = 0xF0000000u;

// QB 32-query blocks per wavefront, WAVES wavefronts: 32 QB WAVES queries
// per workgroup.
template <int QB, int WAVES>
struct WideCfg {
  static constexpr int kTileQ = 32 * QB * WAVES;
  static constexpr int kThreads = 64 * WAVES;
  static constexpr int kDma = kTileB / 1024 / WAVES;  // 1 KB K (and V) copies per wave and tile
  static constexpr int kOps = 2 * kDma;               // K/V copies per wave and tile
  static constexpr int kKeysPerWave = kTileK / WAVES;
  static_assert(kDma * WAVES * 1024 == kTileB && kKeysPerWave == 4 * kDma, "copy split");
};

template <int QB, int WAVES>
__global__ __launch_bounds__(64 * WAVES, 1) void attention_wide_kernel(PvArgs pa) {
  using C = WideCfg<QB, WAVES>;

  __shared__ __attribute__((aligned(1024))) char ring[kWdStages * kStageB];
  __shared__ __attribute__((aligned(16))) char slot_ring[WAVES * 4 * kWdSlotB];
  const AttnArgs& a = pa.a;
  const int splits = pa.splits;

  // XCD-contiguous, head-major order of (head, query tile, key split)
  const int n_tiles_q = a.tile_start[a.batch];
  int h, tile, split;
  {
    const int nb = gridDim.x, i = blockIdx.x;
    const int q8 = nb >> 3, r8 = nb & 7, x = i & 7;
    const int t = x * q8 + min(x, r8) + (i >> 3);
    h = t / (n_tiles_q * splits);
    const int rem = t - h * n_tiles_q * splits;
    tile = rem / splits;
    split = rem - tile * splits;
  }
  int b = 0;
  {
    int lo = 0, hi = a.batch - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (a.tile_start[mid] <= tile) lo = mid; else hi = mid - 1;
    }
    b = lo;
  }
  const int g = h / (a.H / a.Hkv);
  const int tid = threadIdx.x, lane = tid & 63, hl = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n_rows = a.row_n[b];
  const int64_t r0 = (int64_t)a.row_start[b] + a.row_lo[b];  // global row of query 0
  const int q0 = (tile - a.tile_start[b]) * C::kTileQ + wave * 32 * QB;
  int qi[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) qi[qb] = q0 + 32 * qb + (lane & 31);
  const bool live = q0 < n_rows;  // wave-uniform: a wave without a valid query only copies
  const int S = a.key_len[b];
  const int n_kt = (S + kTileK - 1) / kTileK;
  const int t_lo = split * n_kt / splits, t_hi = (split + 1) * n_kt / splits;

  // query fragments of the 32-query blocks: Q[q][16 s + 8 hl .. +7]
  bf16x8 qf[QB][8];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const bool ok = qi[qb] < n_rows;
    const int64_t qrow = ok ? r0 + qi[qb] : 0;
    const bf16* qp = a.q + qrow * a.q_ld + h * kDh + hl * 8;
#pragma unroll
    for (int s2 = 0; s2 < 8; ++s2) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (ok) v = *reinterpret_cast<const u32x4*>(qp + s2 * 16);
      qf[qb][s2] = __builtin_bit_cast(bf16x8, v);
    }
  }

  const uint32_t pool_bytes = (uint32_t)(a.n_slots * a.pool_ld * 2);  // < 2^31 (host check)
  const rsrc_words kres = buffer_words(a.k_pool, pool_bytes);
  const rsrc_words vres = buffer_words(a.v_pool, pool_bytes);
  const rsrc_words sres = buffer_words(a.slots + a.key_start[b], (uint32_t)S * 4u);
  const int pch = lane & 15;
  const uint32_t head_b = (uint32_t)g * kRowB;
  const uint32_t ld_b = (uint32_t)a.pool_ld * 2u;
  char* const my_slots = slot_ring + wave * 4 * kWdSlotB;

  // the slot indices of tile t (all 64 keys) into this wave's entry t % 4
  auto issue_slots = [&](int t) {
    dma4_asm(sres, (uint32_t)(t * kTileK + lane) * 4u, my_slots + (t & 3) * kWdSlotB);
  };
  // K and V rows of tile t into stage t % 4: this lane's keys (64 / WAVES)
  // wave + 4 i + lane / 16, chunk lane % 16 (K chunks XOR-swizzled by row & 15, V by
  // 2 (row & 3)); reads the tile's slot indices from LDS
  auto kv_offsets = [&](int t, uint32_t (&off)[C::kDma]) {
    const char* sl = my_slots + (t & 3) * kWdSlotB;
#pragma unroll
    for (int i = 0; i < C::kDma; ++i) {
      const int kk = wave * C::kKeysPerWave + 4 * i + (lane >> 4);
      const int key = t * kTileK + kk;
      const int slot = *reinterpret_cast<const int*>(sl + kk * 4);
      const bool ok = key < S && slot >= 0 && slot < a.n_slots;
      off[i] = ok ? (uint32_t)slot * ld_b + head_b : kWdAbsent;
    }
  };
  auto kv_issue = [&](int t, const uint32_t (&off)[C::kDma], int i) {
    char* st = ring + (t & 3) * kStageB;
    const int r = (wave * C::kKeysPerWave + 4 * i + (lane >> 4)) & (kTileK - 1);
    const int ck = pch ^ (r & 15), cv = pch ^ ((r & 3) << 1);
    const int dst = (wave * C::kDma + i) * 1024;
    dma16_asm(kres, off[i] + ck * 16, st + dst);
    dma16_asm(vres, off[i] + cv * 16, st + kTileB + dst);
  };
  auto issue_kv = [&](int t) {
    uint32_t off[C::kDma];
    kv_offsets(t, off);
#pragma unroll
    for (int i = 0; i < C::kDma; ++i) kv_issue(t, off, i);
  };

  const float scale = kLog2e * rsqrtf((float)kDh);
  const int krow = key_perm(lane & 31);
  const int k_row_off = krow * kRowB;
  const int k_sw = krow & 15;
  const int vgrp = lane >> 4, gi = lane & 15;
  const int v_key = 8 * (vgrp >> 1) + (gi >> 2);
  const int v_chunk_lo = 2 * (vgrp & 1) + ((gi & 3) >> 1);
  const int v_byte = (gi & 1) * 8;
  const int v_sw = (gi >> 2) << 1;

  // S^T of tile t for both query blocks: st[qb][kb], register r of key block
  // kb holding key 32 kb + 16 (r / 8) + 8 hl + r % 8 of the tile
  auto scores = [&](int t, f32x16 (&st)[QB][2]) {
    const char* ks = ring + (t & 3) * kStageB;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int r = 0; r < 16; ++r) st[qb][kb][r] = 0.f;
#pragma unroll
      for (int s2 = 0; s2 < 8; ++s2) {
        const bf16x8 kf =
            *reinterpret_cast<const bf16x8*>(ks + kb * 32 * kRowB + k_row_off + (((2 * s2 + hl) ^ k_sw) << 4));
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) st[qb][kb] = mfma32x32x16(kf, qf[qb][s2], st[qb][kb]);
      }
    }
  };
  // keys of tile t past the end: -inf; returns the scaled row maxima
  auto row_max = [&](int t, f32x16 (&st)[QB][2], float (&mx)[QB]) {
    const int kt0 = t * kTileK;
    const uint64_t drop = kt0 + kTileK <= S ? 0ull : ~0ull << (S - kt0);
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      float m = -INFINITY;
      if (drop == 0ull) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) m = fmaxf(m, st[qb][kb][r]);
      } else {
        const uint32_t dw[2] = {(uint32_t)drop >> (8 * hl), (uint32_t)(drop >> 32) >> (8 * hl)};
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            st[qb][kb][r] = (dw[kb] >> (16 * (r >> 3) + (r & 7))) & 1u ? -INFINITY : st[qb][kb][r];
            m = fmaxf(m, st[qb][kb][r]);
          }
      }
      mx[qb] = fmaxf(m, __shfl_xor(m, 32)) * scale;
    }
  };

  f32x16 o_acc[QB][4];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb)
#pragma unroll
    for (int d = 0; d < 4; ++d)
#pragma unroll
      for (int r = 0; r < 16; ++r) o_acc[qb][d][r] = 0.f;
  float m_run[QB], l_part[QB], lse_aff2[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    m_run[qb] = -INFINITY;
    l_part[qb] = 0.f;
    lse_aff2[qb] = -INFINITY;
  }
  const int aff_end = min(a.aff_t1, t_hi);
  // moves the running max of a block whose tile maximum exceeds it by more
  // than 2^8, rescaling what has been accumulated
  auto rescale = [&](const float (&mx)[QB]) {
    bool any = false;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) any |= mx[qb] > m_run[qb] + 8.f;
    if (__builtin_amdgcn_ballot_w64(any)) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        const bool bp = mx[qb] > m_run[qb] + 8.f;
        const float m_new = bp ? mx[qb] : m_run[qb];
        const float alpha = __builtin_amdgcn_exp2f(m_run[qb] - m_new);
        m_run[qb] = m_new;
        l_part[qb] *= alpha;
#pragma unroll
        for (int d = 0; d < 4; ++d)
#pragma unroll
          for (int r = 0; r < 16; ++r) o_acc[qb][d][r] *= alpha;
      }
    }
  };

  constexpr int kOps = C::kOps;
  f32x16 st_a[QB][2], st_b[QB][2];
  float mx[QB];
  if (t_lo < t_hi) {
    // prologue: slot indices of the first three tiles, then their K/V rows
    issue_slots(t_lo);
    issue_slots(t_lo + 1);
    issue_slots(t_lo + 2);
    wait_vm_asm<2>();
    issue_kv(t_lo);
    wait_vm_asm<kOps + 1>();
    issue_kv(t_lo + 1);
    wait_vm_asm<2 * kOps>();
    issue_slots(t_lo + 3);
    issue_kv(t_lo + 2);
    wait_vm_asm<2 * kOps + 1>();  // tile t_lo has landed in this wave
    bare_barrier();
    if (live) {
      scores(t_lo, st_a);
      row_max(t_lo, st_a, mx);
      rescale(mx);
    }
  }
  // one iteration: P(t) from cur, S(t+1) into nxt, O += V P(t), max of t+1
  auto step = [&](int t, f32x16 (&cur)[QB][2], f32x16 (&nxt)[QB][2]) {
    wait_vm_asm<kOps>();  // tile t+1 and the slot indices of tile t+3 have landed in this wave
    bare_barrier();       // ... in every wave, and every wave is done with tile t-1
    if (!live) {
      issue_slots(t + 4);
      issue_kv(t + 3);  // into the stage of tile t-1
      return;
    }
    // The iteration is laid out by hand in chunks fenced against the
    // scheduler: 16 chunks of one S(t+1) MFMA (K fragment read kWdKAhead
    // chunks ahead) with two of tile t's exponentials, then 16 chunks of one
    // P V MFMA (V fragment read kWdVAhead chunks ahead) with the maxima of two
    // of tile t+1's logits.  The empty asm statements keep the running sum and
    // maximum inside their chunk (without them the compiler sinks the adds
    // and maxima past the MFMAs).  Every accumulator sees the same MFMA
    // sequence as in attention_pv_kernel.
    const char* ks = ring + ((t + 1) & 3) * kStageB;
    const char* vs = ring + (t & 3) * kStageB + kTileB;
    auto kfrag = [&](int i) {
      const int kb = i >> 3, s2 = i & 7;
      return *reinterpret_cast<const bf16x8*>(ks + kb * 32 * kRowB + k_row_off + (((2 * s2 + hl) ^ k_sw) << 4));
    };
    auto vfrag = [&](int i) {
      const int kb = i >> 3, g2 = (i >> 2) & 1, d = i & 3;
      const int row0 = kb * 32 + g2 * 16 + v_key;
      const int off = ((4 * d + v_chunk_lo) ^ v_sw) * 16 + v_byte;
      const v4i16 lo = ds_read_tr16(vs + row0 * kRowB + off);
      const v4i16 hi = ds_read_tr16(vs + (row0 + 4) * kRowB + off);
      return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
    };
    bf16x8 pb[QB][2][2];
    float psum[QB];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      psum[qb] = 0.f;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) nxt[qb][kb][r] = 0.f;
    }
    bf16x8 kf[kWdKAhead + 1];
#pragma unroll
    for (int i = 0; i < kWdKAhead; ++i) kf[i] = kfrag(i);
    bf16x8 vf[kWdVAhead + 1];
    uint32_t koff[C::kDma];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      // the copies of tile t+3 (into the stage of tile t-1), spread over
      // the first chunks: slot indices of tile t+4, offsets, K/V rows
      if (i == 0) issue_slots(t + 4);
      if (i == 1) kv_offsets(t + 3, koff);
#pragma unroll
      for (int j = 0; j < C::kDma; ++j)
        if (i == 3 + 2 * j) kv_issue(t + 3, koff, j);
      if (i + kWdKAhead < 16) kf[(i + kWdKAhead) % (kWdKAhead + 1)] = kfrag(i + kWdKAhead);
      if (i >= 16 - kWdVAhead) vf[i - (16 - kWdVAhead)] = vfrag(i - (16 - kWdVAhead));
      const int kb = i >> 3, s2 = i & 7;
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) nxt[qb][kb] = mfma32x32x16(kf[i % (kWdKAhead + 1)], qf[qb][s2], nxt[qb][kb]);
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const int e = 2 * i + u, ekb = e >> 4, r = e & 15;
          const float x = __builtin_amdgcn_exp2f(fmaf(cur[qb][ekb][r], scale, -m_run[qb]));
          psum[qb] += x;
          pb[qb][ekb][r >> 3][r & 7] = (bf16)x;
        }
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) asm volatile("" ::"v"(psum[qb]));
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      l_part[qb] += psum[qb];
      if (t + 1 == aff_end) lse_aff2[qb] = m_run[qb] + __log2f(l_part[qb] + __shfl_xor(l_part[qb], 32));
      mx[qb] = -INFINITY;
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      if (i + kWdVAhead < 16) vf[(i + kWdVAhead) % (kWdVAhead + 1)] = vfrag(i + kWdVAhead);
      const int kb = i >> 3, g2 = (i >> 2) & 1, d = i & 3;
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) o_acc[qb][d] = mfma32x32x16(vf[i % (kWdVAhead + 1)], pb[qb][kb][g2], o_acc[qb][d]);
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        mx[qb] = fmaxf(mx[qb], fmaxf(nxt[qb][i >> 3][2 * (i & 7)], nxt[qb][i >> 3][2 * (i & 7) + 1]));
        asm volatile("" ::"v"(mx[qb]));
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    if (t + 1 < t_hi) {
      if ((t + 2) * kTileK > S) {
        row_max(t + 1, nxt, mx);
      } else {
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) mx[qb] = fmaxf(mx[qb], __shfl_xor(mx[qb], 32)) * scale;
      }
      rescale(mx);
    }
  };
  int t = t_lo;
  for (; t + 1 < t_hi; t += 2) {
    step(t, st_a, st_b);
    step(t + 1, st_b, st_a);
  }
  if (t < t_hi) step(t, st_a, st_b);
  // every copy this wave issued has landed before the workgroup ends
  wait_vm_asm<0>();

  if (!live) return;
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const float l_tot = l_part[qb] + __shfl_xor(l_part[qb], 32);
    if (qi[qb] >= n_rows) continue;
    const int64_t row = r0 + qi[qb];
    if (splits > 1) {
      const int64_t prow = (int64_t)a.row_start[a.batch];
      float* po = pa.part_o + (((int64_t)split * prow + row) * a.H + h) * kDh;
#pragma unroll
      for (int d = 0; d < 4; ++d)
#pragma unroll
        for (int gq = 0; gq < 4; ++gq) {
          const f32x4 v = {o_acc[qb][d][4 * gq], o_acc[qb][d][4 * gq + 1], o_acc[qb][d][4 * gq + 2],
                           o_acc[qb][d][4 * gq + 3]};
          *reinterpret_cast<f32x4*>(po + d * 32 + 8 * gq + 4 * hl) = v;
        }
      if (hl == 0) {
        float* pm = pa.part_ml + (((int64_t)split * prow + row) * a.H + h) * 2;
        pm[0] = m_run[qb];
        pm[1] = l_tot;
        if (pa.part_aff) pa.part_aff[((int64_t)split * prow + row) * a.H + h] = lse_aff2[qb];
      }
      continue;
    }
    if (a.lse && hl == 0) a.lse[row * a.H + h] = (m_run[qb] + __log2f(l_tot)) * kLn2;
    if (a.lse_aff && hl == 0) a.lse_aff[row * a.H + h] = lse_aff2[qb] * kLn2;
    const float inv = 1.f / l_tot;
    bf16* op = a.out + row * (int64_t)a.H * kDh + (int64_t)h * kDh;
#pragma unroll
    for (int d = 0; d < 4; ++d)
#pragma unroll
      for (int gq = 0; gq < 4; ++gq) {
        bf16x4 w;
#pragma unroll
        for (int j = 0; j < 4; ++j) w[j] = (bf16)(o_acc[qb][d][4 * gq + j] * inv);
        *reinterpret_cast<bf16x4*>(op + d * 32 + 8 * gq + 4 * hl) = w;
      }
  }
}

}  // namespace


// Key splits for the read-slot attention.  Cost in 64-key tiles of one
// 128-query workgroup (about 1 us each): rounds of `slots` resident
// workgroups times the tiles per split times the cost of one tile, plus the
// merge traffic (each split's fp32 O and (m, l), and extra_b more bytes per
// (row, head), written and read back at about 6 TB/s).  The partials must
// fit in part_bytes.  Returns the splits; *cost receives the estimate.
static int attention_splits(int n_wg, int slots, double tile_cost, int n_kt, int64_t rows, int H,
                            size_t part_bytes, int extra_b, double* cost) {
  const int64_t per_split = rows * H * (kDh * 4 + 8 + extra_b);
  int best = 1;
  double best_cost = 1e30;
  for (int s = 1; s <= 8 && s <= n_kt; ++s) {
    if (s > 1 && (size_t)(per_split * s) > part_bytes) break;
    const double rounds = (double)((n_wg * s + slots - 1) / slots);
    const double tiles = (double)((n_kt + s - 1) / s);
    // merge: 2 x per_split x s bytes at ~6 TB/s, one 64-key tile of a workgroup ~1 us
    const double merge = s > 1 ? 2.0 * per_split * s / 6e12 / 1e-6 : 0.0;
    const double c = rounds * tiles * tile_cost + merge;
    if (c < best_cost) {
      best_cost = c;
      best = s;
    }
  }
  *cost = best_cost;
  return best;
}

// One 64-key tile of a 256-query workgroup of attention_wide_kernel (one
// per CU), in units of a 128-query workgroup's tile (two per CU), measured
// on the serving shapes (40% against 36.5% of the bf16 peak).
constexpr double kWideTileCost = 0.9;
constexpr int kWideQB = 1, kWideWaves = 8;
using WideQ = WideCfg<kWideQB, kWideWaves>;

hipError_t launch_attention_bf16(const Ragged& rg, int H, int Hkv, const void* q,
                                 const int32_t* read_slots, const void* k_pool, const void* v_pool,
                                 int64_t pool_ld, int64_t n_slots, void* out, float* lse,
                                 float* part, size_t part_bytes, hipStream_t s, float* lse_aff, int aff_begin,
                                 int aff_len, bool* aff_done) {
  if (aff_done) *aff_done = false;
  // the affix log-sum-exp rides along where the affix keys come first, in
  // whole key tiles (under key splits through one more fp32 partial per
  // split, row and head)
  const bool want_aff = lse_aff && aff_len > 0 && aff_begin == 0 && aff_len % kTileK == 0;
  PvArgs pa = {};
  AttnArgs& a = pa.a;
  a.q = (const bf16*)q;
  a.q_ld = (int64_t)H * kDh;
  a.q_n_rows = rg.cu_rows[rg.batch];
  a.q_idx = nullptr;
  a.slots = read_slots;
  a.k_pool = (const bf16*)k_pool;
  a.v_pool = (const bf16*)v_pool;
  a.pool_ld = pool_ld;
  a.n_slots = n_slots;
  a.out = (bf16*)out;
  a.lse = lse;
  a.H = H;
  a.Hkv = Hkv;
  a.batch = rg.batch;
  for (int b = 0; b <= rg.batch; ++b) {
    a.row_start[b] = rg.cu_rows[b];
    a.key_start[b] = rg.cu_keys[b];
  }
  const int64_t rows = rg.cu_rows[rg.batch];
  if (rows == 0) return hipSuccess;
  int tiles = 0, tiles_w = 0, max_kt = 0, full_w = 0, rem_n = 0;
  for (int b = 0; b < rg.batch; ++b) {
    a.key_len[b] = rg.cu_keys[b + 1] - rg.cu_keys[b];
    const int nr = a.row_start[b + 1] - a.row_start[b];
    a.row_lo[b] = 0;
    a.row_n[b] = nr;
    tiles += (nr + kPvTileQ - 1) / kPvTileQ;
    tiles_w += (nr + WideQ::kTileQ - 1) / WideQ::kTileQ;
    full_w += nr / WideQ::kTileQ;
    rem_n += (nr % WideQ::kTileQ + kPvTileQ - 1) / kPvTileQ;
    max_kt = std::max(max_kt, (a.key_len[b] + kTileK - 1) / kTileK);
  }
  if (tiles == 0) return hipSuccess;
  const size_t pbytes = part ? part_bytes : 0;
  double cost_n = 0.0, cost_w = 0.0;
  const int aff_b = want_aff ? 4 : 0;
  const int splits_n = attention_splits(tiles * H, 512, 1.0, max_kt, rows, H, pbytes, aff_b, &cost_n);
  const int splits_w = attention_splits(tiles_w * H, 256, kWideTileCost, max_kt, rows, H, pbytes, aff_b, &cost_w);
  const bool wide_ok = (uint64_t)n_slots * (uint64_t)pool_ld * 2u <= (uint64_t)kWdAbsent;
  // the wide kernel wherever the cost model prefers it, below one round of
  // CUs too (C2's refresh: 96 query tiles x 2 key splits, attention 10%
  // faster than the 128-query kernel's 384 workgroups)
  const bool wide = wide_ok && cost_w < cost_n;
  // split: each request's whole 256-row tiles on the wide kernel and its
  // last partial tile (in 128-row tiles) on the two-per-CU kernel, one launch
  // each, no key splits (the merge kernel would cover every row)
  const double cost_split = (double)((full_w * H + 255) / 256) * max_kt * kWideTileCost +
                            (double)((rem_n * H + 511) / 512) * max_kt;
  auto take_aff = [&]() {
    if (!want_aff) return;
    a.lse_aff = lse_aff;
    a.aff_t1 = aff_len / kTileK;
    if (aff_done) *aff_done = true;
  };
  if (wide_ok && full_w * H >= 256 && rem_n > 0 && cost_split < std::min(cost_w, cost_n)) {
    pa.splits = 1;
    take_aff();
    int acc = 0;
    for (int b = 0; b < rg.batch; ++b) {
      const int nr = a.row_start[b + 1] - a.row_start[b];
      a.row_n[b] = nr - nr % WideQ::kTileQ;
      a.tile_start[b] = acc;
      acc += a.row_n[b] / WideQ::kTileQ;
    }
    a.tile_start[rg.batch] = acc;
    hipLaunchKernelGGL((attention_wide_kernel<kWideQB, kWideWaves>), dim3(acc * H), dim3(WideQ::kThreads), 0, s, pa);
    acc = 0;
    for (int b = 0; b < rg.batch; ++b) {
      const int nr = a.row_start[b + 1] - a.row_start[b];
      a.row_lo[b] = nr - nr % WideQ::kTileQ;
      a.row_n[b] = nr % WideQ::kTileQ;
      a.tile_start[b] = acc;
      acc += (a.row_n[b] + kPvTileQ - 1) / kPvTileQ;
    }
    a.tile_start[rg.batch] = acc;
    hipLaunchKernelGGL(attention_pv_kernel<false>, dim3(acc * H), dim3(kPvThreads), 0, s, pa);
    return hipGetLastError();
  }
  const int tq = wide ? WideQ::kTileQ : kPvTileQ;
  const int splits = wide ? splits_w : splits_n;
  int acc_tiles = 0;
  for (int b = 0; b < rg.batch; ++b) {
    a.tile_start[b] = acc_tiles;
    acc_tiles += (a.row_start[b + 1] - a.row_start[b] + tq - 1) / tq;
  }
  a.tile_start[rg.batch] = acc_tiles;
  pa.splits = splits;
  take_aff();
  pa.part_o = part;
  pa.part_ml = part ? part + (size_t)splits * rows * H * kDh : nullptr;
  if (splits > 1 && a.lse_aff) pa.part_aff = pa.part_ml + (size_t)splits * rows * H * 2;
  if (wide)
    hipLaunchKernelGGL((attention_wide_kernel<kWideQB, kWideWaves>), dim3(acc_tiles * H * splits),
                       dim3(WideQ::kThreads), 0, s, pa);
  else
    hipLaunchKernelGGL(attention_pv_kernel<false>, dim3(acc_tiles * H * splits), dim3(kPvThreads), 0, s, pa);
  if (splits > 1) {
    const int64_t pairs = rows * H;
    hipLaunchKernelGGL(attention_merge_kernel, dim3((unsigned)((pairs + 7) / 8)), dim3(256), 0, s,
                       (const float*)pa.part_o, (const float*)pa.part_ml, splits, rows, H, (bf16*)out, lse,
                       (const float*)pa.part_aff, pa.part_aff ? lse_aff : nullptr);
  }
  return hipGetLastError();
}

// Key masks of the decode step's shared pass: bit j % 64 of word
// [b][j / 64] is set iff affix-local index j is one of request b's anchors
// (those positions are read from the request's private slots instead).  One
// workgroup per request builds its words in LDS.
__global__ __launch_bounds__(256) void anchor_mask_kernel(const int32_t* __restrict__ anchors, int k, int L,
                                                          int n_words, uint64_t* __restrict__ mask) {
  __shared__ unsigned long long words[1024];
  const int b = blockIdx.x;
  for (int i = threadIdx.x; i < n_words; i += 256) words[i] = 0ull;
  __syncthreads();
  for (int i = threadIdx.x; i < k; i += 256) {
    const int j = anchors[(int64_t)b * k + i];
    if (j >= 0 && j < L) atomicOr(&words[j >> 6], 1ull << (j & 63));
  }
  __syncthreads();
  for (int i = threadIdx.x; i < n_words; i += 256) mask[(int64_t)b * n_words + i] = words[i];
}

// Decode-step attention over a view made of the shared affix (minus each
// request's anchors) and each request's private keys.  Pass 1 takes the
// queries of all requests together against the shared affix keys, so each
// K/V tile of the affix is read once per 128 queries instead of once per
// request; pass 2 takes each request's queries against its private keys.
// Both write (O, max, sum) partials, which the merge kernel combines.
hipError_t launch_attention_decode_bf16(int batch, int rows_per_req, int H, int Hkv, const void* q,
                                        const int32_t* affix_slots, int L, const int32_t* anchors, int k,
                                        const int32_t* private_slots, int private_len, const void* k_pool,
                                        const void* v_pool, int64_t pool_ld, int64_t n_slots, void* out,
                                        uint64_t* mask, float* part, size_t part_bytes, hipStream_t s) {
  const int64_t rows = (int64_t)batch * rows_per_req;
  if (rows == 0) return hipSuccess;
  const bool shared = L > k;  // some affix position is read from the shared slots
  const int64_t per_split = rows * H * (kDh * 4 + 8);
  const int q_tiles_all = (int)((rows + kPvTileQ - 1) / kPvTileQ);
  const int q_tiles_req = (rows_per_req + kPvTileQ - 1) / kPvTileQ;
  const int n_kt_shared = (L + kTileK - 1) / kTileK;
  if ((size_t)per_split * (shared ? 2 : 1) > part_bytes) return hipErrorInvalidValue;
  const int sp_priv = 1;
  double cost_unused = 0.0;
  const int sp_shared = shared ? attention_splits(q_tiles_all * H, 512, 1.0, n_kt_shared, rows, H,
                                                  part_bytes - (size_t)per_split * sp_priv, 0, &cost_unused)
                               : 0;
  const int total = sp_shared + sp_priv;

  auto common = [&](PvArgs& pa) {
    AttnArgs& a = pa.a;
    a.q = (const bf16*)q;
    a.q_ld = (int64_t)H * kDh;
    a.q_n_rows = rows;
    a.q_idx = nullptr;
    a.k_pool = (const bf16*)k_pool;
    a.v_pool = (const bf16*)v_pool;
    a.pool_ld = pool_ld;
    a.n_slots = n_slots;
    a.out = (bf16*)out;
    a.lse = nullptr;
    a.H = H;
    a.Hkv = Hkv;
    pa.part_o = part;
    pa.part_ml = part + (size_t)total * rows * H * kDh;
    pa.partial = 1;
    pa.part_rows = rows;
  };
  if (shared) {
    hipLaunchKernelGGL(anchor_mask_kernel, dim3(batch), dim3(256), 0, s, anchors, k, L, n_kt_shared, mask);
    PvArgs pa = {};
    common(pa);
    AttnArgs& a = pa.a;
    a.slots = affix_slots;
    a.batch = 1;
    a.row_start[0] = 0;
    a.row_start[1] = (int)rows;
    a.row_lo[0] = 0;
    a.row_n[0] = (int)rows;
    a.key_start[0] = 0;
    a.key_start[1] = L;
    a.key_len[0] = L;
    a.tile_start[0] = 0;
    a.tile_start[1] = q_tiles_all;
    pa.splits = sp_shared;
    pa.split_base = 0;
    pa.key_mask = mask;
    pa.mask_tiles = n_kt_shared;
    pa.mask_rows = rows_per_req;
    hipLaunchKernelGGL(attention_pv_kernel<true>, dim3(q_tiles_all * H * sp_shared), dim3(kPvThreads), 0, s, pa);
  }
  {
    PvArgs pa = {};
    common(pa);
    AttnArgs& a = pa.a;
    a.slots = private_slots;
    a.batch = batch;
    for (int b = 0; b <= batch; ++b) {
      a.row_start[b] = b * rows_per_req;
      if (b < batch) {
        a.row_lo[b] = 0;
        a.row_n[b] = rows_per_req;
      }
      a.key_start[b] = b * private_len;
      a.tile_start[b] = b * q_tiles_req;
    }
    for (int b = 0; b < batch; ++b) a.key_len[b] = private_len;
    pa.splits = sp_priv;
    pa.split_base = sp_shared;
    hipLaunchKernelGGL(attention_pv_kernel<false>, dim3(batch * q_tiles_req * H * sp_priv), dim3(kPvThreads), 0, s,
                       pa);
  }
  const int64_t pairs = rows * H;
  hipLaunchKernelGGL(attention_merge_kernel, dim3((unsigned)((pairs + 7) / 8)), dim3(256), 0, s, (const float*)part,
                     (const float*)(part + (size_t)total * rows * H * kDh), total, rows, H, (bf16*)out, nullptr,
                     nullptr, nullptr);
  return hipGetLastError();
}


}  // namespace acache
