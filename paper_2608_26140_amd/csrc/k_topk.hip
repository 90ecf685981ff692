// Exact top-K anchor selection (Section 3.2, Eq. 6), one workgroup per
// request.
//
// Scores become order-preserving 32-bit keys (-0 is folded onto +0, NaN maps
// below -inf).  A 4-pass, 8-bit-digit radix select over the keys in LDS finds
// the K-th largest key T and how many of the K winners must be taken from the
// keys equal to T.  A stable compaction in index order then writes the
// winners ascending: every key above T, and the lowest-index keys equal to T.
// The result depends only on the input bits.
#include "device.h"
#include "internal.h"

namespace acache {

namespace {

constexpr int kTopkThreads = 1024;
constexpr int kTopkWaves = kTopkThreads / 64;

// Exclusive prefix sum of one int per thread over the workgroup.
__device__ int block_excl_scan(int v, int* wsum) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int incl = wave_incl_scan(v);
  if (lane == 63) wsum[wave] = incl;
  __syncthreads();
  if (wave == 0) {
    int t = lane < kTopkWaves ? wsum[lane] : 0;
    const int ti = wave_incl_scan(t);
    if (lane < kTopkWaves) wsum[lane] = ti - t;
  }
  __syncthreads();
  const int r = wsum[wave] + incl - v;
  __syncthreads();
  return r;
}

__global__ __launch_bounds__(kTopkThreads) void topk_kernel(const uint32_t* __restrict__ scores, int L,
                                                            int k, int32_t* __restrict__ out) {
  extern __shared__ uint32_t keys[];
  __shared__ int hist[256];
  __shared__ int wsum[kTopkWaves];
  __shared__ int sel_digit, sel_above;
  const int b = blockIdx.x;
  const uint32_t* s = scores + (int64_t)b * L;
  for (int j = threadIdx.x; j < L; j += kTopkThreads) keys[j] = order_key(s[j]);

  uint32_t prefix = 0u, pmask = 0u;
  int remaining = k;  // winners still to place at or below the current prefix
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    if (threadIdx.x < 256) hist[threadIdx.x] = 0;
    __syncthreads();
    for (int j = threadIdx.x; j < L; j += kTopkThreads) {
      const uint32_t key = keys[j];
      if ((key & pmask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1);
    }
    __syncthreads();
    if (threadIdx.x < 64) {
      // lane l covers digits 255-4l .. 252-4l, highest first
      const int lane = threadIdx.x;
      int c[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) c[q] = hist[255 - 4 * lane - q];
      const int tot = c[0] + c[1] + c[2] + c[3];
      int before = wave_incl_scan(tot) - tot;  // keys in higher digits
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (before < remaining && before + c[q] >= remaining) {
          sel_digit = 255 - 4 * lane - q;
          sel_above = before;
        }
        before += c[q];
      }
    }
    __syncthreads();
    prefix |= (uint32_t)sel_digit << shift;
    pmask |= 0xFFu << shift;
    remaining -= sel_above;
    __syncthreads();
  }
  const uint32_t T = prefix;
  const int need_eq = remaining;  // winners equal to T, lowest indices first

  // contiguous chunk per thread keeps index order
  const int per = (L + kTopkThreads - 1) / kTopkThreads;
  const int j0 = min(L, (int)threadIdx.x * per), j1 = min(L, j0 + per);
  int n_eq = 0;
  for (int j = j0; j < j1; ++j) n_eq += keys[j] == T;
  const int eq_before = block_excl_scan(n_eq, wsum);
  int n_sel = 0, e = eq_before;
  for (int j = j0; j < j1; ++j) {
    const uint32_t key = keys[j];
    if (key > T) ++n_sel;
    else if (key == T) { n_sel += e < need_eq; ++e; }
  }
  int o = block_excl_scan(n_sel, wsum);
  e = eq_before;
  int32_t* ob = out + (int64_t)b * k;
  for (int j = j0; j < j1; ++j) {
    const uint32_t key = keys[j];
    bool take = key > T;
    if (key == T) { take = e < need_eq; ++e; }
    if (take && o < k) ob[o++] = j;
  }
}

}  // namespace

hipError_t launch_topk(const float* scores, int batch, int L, int k, int32_t* out, hipStream_t s) {
  hipLaunchKernelGGL(topk_kernel, dim3(batch), dim3(kTopkThreads), (size_t)L * sizeof(uint32_t), s,
                     (const uint32_t*)scores, L, k, out);
  return hipGetLastError();
}

}  // namespace acache
