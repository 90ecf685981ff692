// Device-side helpers shared by the gfx950 kernels of the selective affix-KV
// recompute path: storage types, MFMA fragment types, wavefront reductions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace acache {

typedef __bf16 bf16;
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ float to_f32(bf16 v) { return (float)v; }
__device__ __forceinline__ float to_f32(float v) { return v; }
template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float v) { return (bf16)v; }
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }

// 32x32x16 bf16 MFMA (gfx950).  Lane l supplies A[l%32][8*(l/32) + j] and
// B[8*(l/32) + j][l%32], j = 0..7; it receives D[8*(r/4) + 4*(l/32) + r%4][l%32]
// in accumulator register r = 0..15.
__device__ __forceinline__ f32x16 mfma32x32x16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// 16-byte global -> LDS copy (global_load_lds_dwordx4): lane l's 16 bytes
// from g land at lds + 16 l, lds being uniform across the wave.  Completion
// is counted by vmcnt.
__device__ __forceinline__ void dma16(const void* g, char* lds) {
  __builtin_amdgcn_global_load_lds(g, (__attribute__((address_space(3))) void*)lds, 16, 0, 0);
}

// Raw buffer resource over [base, base + bytes) (gfx9 descriptor: stride 0,
// num_records in bytes).  Loads through it past the end return zeros.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}
// 16-byte buffer -> LDS copy (buffer_load_dwordx4 ... lds): lane l's 16 bytes
// at voff + soff land at lds + 16 l (lds uniform across the wave); soff is
// a wave-uniform byte offset held in an SGPR.  Completion is counted by vmcnt.
__device__ __forceinline__ void dma16_buf(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff, char* lds) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds, 16, voff, soff, 0, 0);
}

// s_waitcnt on one counter, the others left at their maximum (gfx9
// encoding: vmcnt in bits 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt field");
  __builtin_amdgcn_s_waitcnt(0x0F70 | (N & 15) | ((N >> 4) << 14));
}
template <int N>
__device__ __forceinline__ void wait_lgkmcnt() {
  static_assert(N >= 0 && N < 16, "lgkmcnt field");
  __builtin_amdgcn_s_waitcnt(0xC07F | (N << 8));
}

// This lane's index in its wavefront, computed where it is called: the
// compiler cannot hoist the asm out of a loop, so nothing derived from the
// lane index has to stay live (or be spilled) across the loop's body.
__device__ __forceinline__ int lane_id_here() {
  int l;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n v_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
  return l;
}

// Workgroup barrier that orders LDS only.  __syncthreads() also waits for
// every outstanding global load, which would include loads in flight to
// LDS for later stages; those are tracked with explicit vmcnt waits.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Workgroup barrier with no fence: the caller has already waited (vmcnt /
// lgkmcnt) for whatever LDS traffic the other waves must see.  The asm's
// memory clobber keeps the compiler from moving memory accesses across it.
__device__ __forceinline__ void bare_barrier() { asm volatile("s_barrier" ::: "memory"); }

// Order-preserving 32-bit key of an fp32 bit pattern: larger float, larger
// key; -0 is folded onto +0 and NaN maps below -inf (key 0).
__device__ __forceinline__ uint32_t order_key(uint32_t u) {
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0u;  // NaN: below everything
  if (u == 0x80000000u) u = 0u;                     // -0 == +0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// sin and cos of a rotary angle given in fp64.  The angle is reduced to
// r = ang - q * pi/2, |r| <= pi/4, in fp64 (the product pos * theta_i is
// exact enough there for any position), then both functions are Taylor
// polynomials in r to degree 11 / 12 (truncation below 1e-9) evaluated in
// fp32, and the quadrant q mod 4 picks signs and swaps.  Unlike the library
// sincos, this has no large-argument path and no scratch table.
__device__ __forceinline__ void rotary_sincos(double ang, float* sn, float* cs) {
  const double q = rint(ang * 0.6366197723675814);  // 2 / pi
  const float r = (float)(ang - q * 1.5707963267948966);
  const float r2 = r * r;
  // sin r = r (1 - r^2/3! (1 - r^2/(4*5) (1 - r^2/(6*7) (1 - r^2/(8*9) (1 - r^2/(10*11))))))
  float ps = 1.f - r2 * (1.f / 110.f);
  ps = 1.f - r2 * (1.f / 72.f) * ps;
  ps = 1.f - r2 * (1.f / 42.f) * ps;
  ps = 1.f - r2 * (1.f / 20.f) * ps;
  ps = 1.f - r2 * (1.f / 6.f) * ps;
  const float s = r * ps;
  // cos r = 1 - r^2/2! (1 - r^2/(3*4) (1 - r^2/(5*6) (1 - r^2/(7*8) (1 - r^2/(9*10) (1 - r^2/(11*12))))))
  float pc = 1.f - r2 * (1.f / 132.f);
  pc = 1.f - r2 * (1.f / 90.f) * pc;
  pc = 1.f - r2 * (1.f / 56.f) * pc;
  pc = 1.f - r2 * (1.f / 30.f) * pc;
  pc = 1.f - r2 * (1.f / 12.f) * pc;
  const float c = 1.f - r2 * 0.5f * pc;
  const int k = (int)((long long)q & 3);
  *sn = k == 0 ? s : k == 1 ? c : k == 2 ? -s : -c;
  *cs = k == 0 ? c : k == 1 ? -s : k == 2 ? -c : s;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
__device__ __forceinline__ int wave_sum_int(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
// Inclusive prefix sum across the 64 lanes of a wavefront.
__device__ __forceinline__ int wave_incl_scan(int v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int t = __shfl_up(v, o);
    if (lane >= o) v += t;
  }
  return v;
}

}  // namespace acache
