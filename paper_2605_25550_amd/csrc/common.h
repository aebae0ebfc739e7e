// Device-side helpers shared by the gfx950 kernels of the DiT step.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ditmi {

typedef uint16_t bf16_t;  // storage type of bfloat16 in memory
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2v __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
// Native 16-byte vector for global/LDS staging (HIP's uint4 is a struct whose
// copies go through memcpy and can keep staging arrays in scratch memory).
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf2f(bf16_t v) { return __uint_as_float(((uint32_t)v) << 16); }

// Round-to-nearest-even float -> bf16 pair packed in one dword (low = a).
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  bf16x2v v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}
__device__ __forceinline__ bf16_t f2bf(float a) {
  __bf16 v = (__bf16)a;
  return __builtin_bit_cast(bf16_t, v);
}

template <typename T> __device__ __forceinline__ float ld_as_float(const T* p, long i);
template <> __device__ __forceinline__ float ld_as_float<float>(const float* p, long i) { return p[i]; }
template <> __device__ __forceinline__ float ld_as_float<bf16_t>(const bf16_t* p, long i) { return bf2f(p[i]); }

// Sum over the 64 lanes: DPP moves combine within each 16-lane row (lane
// pairs, quads, half-row mirror, row mirror), then the four row sums are read
// as scalars.  No LDS-crossbar permutes; every lane receives the total.
template <int CTRL>
__device__ __forceinline__ float dpp_move(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_move<0xB1>(v);   // quad_perm [1,0,3,2]
  v += dpp_move<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp_move<0x141>(v);  // row_half_mirror
  v += dpp_move<0x140>(v);  // row_mirror: each lane holds its row's sum
  const int b = __float_as_int(v);
  return (__int_as_float(__builtin_amdgcn_readlane(b, 0)) + __int_as_float(__builtin_amdgcn_readlane(b, 16))) +
         (__int_as_float(__builtin_amdgcn_readlane(b, 32)) + __int_as_float(__builtin_amdgcn_readlane(b, 48)));
}

// n / d for 0 <= n < 2^24, d >= 1 and a quotient below 2^22, given
// inv = 1.0f / d (correctly rounded): the float estimate is within one of the
// quotient, and the two integer corrections make it exact.  Cheaper than the
// integer division sequence for a runtime divisor.
__device__ __forceinline__ int div_exact(int n, int d, float inv) {
  int q = (int)((float)n * inv);
  q -= q * d > n ? 1 : 0;
  q += (q + 1) * d <= n ? 1 : 0;
  return q;
}

// max / sum of v over lanes l and l ^ 32.  v_permlane32_swap exchanges the
// upper half of its first operand with the lower half of its second; with
// both operands v, the two results are {own, partner} in some order, which is
// all a symmetric combine needs.
__device__ __forceinline__ float max_halves(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_halves(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// tanh-approximated GELU; tanh(z) = 1 - 2 / (exp(2z) + 1).
// tanh-GELU: 0.5 u (1 + tanh z) with z = sqrt(2/pi) (u + 0.044715 u^3), in the
// equivalent form u / (1 + exp(-2z)) = u * rcp(1 + exp2(u (c1 + c2 u^2))),
// c1 = -2 log2(e) sqrt(2/pi), c2 = 0.044715 c1.  v_rcp_f32 is within 1 ulp,
// far below the bf16 rounding of the GELU output (and the fp32 path's
// tolerance); exp2 overflow to +inf gives the exact limit 0.
__device__ __forceinline__ float gelu_tanh(float u) {
  const float c1 = -2.30220819814f;           // -2 * log2(e) * sqrt(2/pi)
  const float c2 = -0.10294323958f;           // 0.044715 * c1
  const float e = __builtin_amdgcn_exp2f(u * fmaf(c2, u * u, c1));
  return u * __builtin_amdgcn_rcpf(1.0f + e);
}

// SiLU z / (1 + exp(-z)) with the hardware reciprocal (within 1 ulp).
__device__ __forceinline__ float silu(float z) {
  return z * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-1.4426950408889634f * z));
}

// Workgroup id -> logical tile id so that consecutive logical tiles land on
// the same XCD (workgroups are dispatched round-robin over the 8 XCDs).
__device__ __forceinline__ int xcd_remap(int i, int n) {
  const int X = 8;
  int q = n / X, r = n % X;
  int xcd = i % X, idx = i / X;
  return xcd < r ? xcd * (q + 1) + idx : r * (q + 1) + (xcd - r) * q + idx;
}

// ---------------------------------------------------------------- LDS DMA
// 32-bit LDS address of a __shared__ object.
__device__ __forceinline__ unsigned lds_address(const void* p) {
  return (unsigned)(size_t)(const __attribute__((address_space(3))) void*)p;
}

// One 16-byte-per-lane DMA from global memory into LDS at (wave-uniform)
// base + 16 * lane.
__device__ __forceinline__ void dma_16(const void* gsrc, unsigned lds_base) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
               :
               : "s"(lds_base), "v"(gsrc)
               : "memory", "m0");
}

// 16 bytes per lane from sbase + voff (sbase wave-uniform) into LDS at
// (wave-uniform) lds_base + 16 * lane.
__device__ __forceinline__ void dma_16s(const void* sbase, unsigned voff, unsigned lds_base) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2"
               :
               : "s"(lds_base), "v"(voff), "s"(sbase)
               : "memory", "m0");
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory");
}

}  // namespace ditmi
