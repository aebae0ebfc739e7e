// Measurement tool (not part of the library): the throughput of a bare loop
// of v_mfma_f32_32x32x16_bf16 on every CU, and the core clock it runs at, for
// operands that are all zero, all one, or pseudo-random bf16 (two random sets
// used alternately, so the multiplier inputs change from one MFMA to the
// next, as in a GEMM).  No memory traffic inside the loop.
//   mfma_probe [iters] [workgroups]
// Each workgroup is 8 waves (two per SIMD, as in the library's 256-row GEMM
// and pipelined attention kernels), each wave issuing 8 independent MFMAs per
// iteration.  The clock is the core cycle counter (s_memtime) over the
// 100 MHz real-time counter (s_memrealtime), read at the start and end of
// each wave's loop and averaged over the waves.  Prints TFLOP/s, % of the
// 2.5 PFLOP/s dense bf16 peak, the clock, and the throughput as % of the
// dense peak at that clock.
#include <hip/hip_runtime.h>
#include <cstdio>
#include <cstdlib>
#include <vector>

#define CK(x)                                                                            \
  do {                                                                                   \
    hipError_t e_ = (x);                                                                 \
    if (e_ != hipSuccess) {                                                              \
      printf("HIP %s line %d\n", hipGetErrorString(e_), __LINE__);                       \
      exit(1);                                                                           \
    }                                                                                    \
  } while (0)

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;

__device__ __forceinline__ __bf16 rnd_bf16(unsigned h) {
  h ^= h >> 15;
  h *= 2246822519u;
  h ^= h >> 13;
  const float z = (float)(h & 0xFFFF) / 32768.0f - 1.0f;  // [-1, 1)
  return (__bf16)z;
}

__global__ __launch_bounds__(512) void mfma_loop(int iters, int mode, float* out, unsigned long long* clk) {
  const int tid = blockIdx.x * 512 + threadIdx.x;
  bf16x8 a0, b0, a1, b1;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const unsigned s = (unsigned)tid * 2654435761u + (unsigned)e * 40503u;
    a0[e] = mode == 0 ? (__bf16)0.0f : mode == 1 ? (__bf16)1.0f : rnd_bf16(s ^ 0x1234567u);
    b0[e] = mode == 0 ? (__bf16)0.0f : mode == 1 ? (__bf16)1.0f : rnd_bf16(s ^ 0x89abcdeu);
    a1[e] = mode == 0 ? (__bf16)0.0f : mode == 1 ? (__bf16)1.0f : rnd_bf16(s ^ 0x2468aceu);
    b1[e] = mode == 0 ? (__bf16)0.0f : mode == 1 ? (__bf16)1.0f : rnd_bf16(s ^ 0x13579bdu);
  }
  f32x16 acc[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) acc[q] = f32x16{};
  const unsigned long long t0 = __builtin_amdgcn_s_memtime(), r0 = __builtin_amdgcn_s_memrealtime();
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int q = 0; q < 8; ++q)
      acc[q] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(q & 1 ? a1 : a0, q & 1 ? b1 : b0, acc[q], 0, 0, 0);
  }
  const unsigned long long t1 = __builtin_amdgcn_s_memtime(), r1 = __builtin_amdgcn_s_memrealtime();
  float s = 0.f;
#pragma unroll
  for (int q = 0; q < 8; ++q)
#pragma unroll
    for (int e = 0; e < 16; ++e) s += acc[q][e];
  out[tid] = s;
  if ((threadIdx.x & 63) == 0) {
    const int w = tid >> 6;
    clk[2 * w] = t1 - t0;
    clk[2 * w + 1] = r1 - r0;
  }
}

int main(int argc, char** argv) {
  const int iters = argc > 1 ? atoi(argv[1]) : 20000;
  const int grid = argc > 2 ? atoi(argv[2]) : 256;
  if (iters < 1 || grid < 1 || grid > 65536) {
    printf("usage: mfma_probe [iters >= 1] [workgroups 1..65536]\n");
    return 1;
  }
  const long threads = (long)grid * 512, waves = threads / 64;
  float* out;
  unsigned long long* clk;
  CK(hipMalloc(&out, threads * sizeof(float)));
  CK(hipMalloc(&clk, waves * 2 * sizeof(unsigned long long)));
  std::vector<unsigned long long> h(waves * 2);
  hipEvent_t e0, e1;
  CK(hipEventCreate(&e0));
  CK(hipEventCreate(&e1));
  const char* names[3] = {"zero", "one", "random"};
  for (int mode = 0; mode < 3; ++mode) {
    hipLaunchKernelGGL(mfma_loop, dim3(grid), dim3(512), 0, 0, iters / 10 + 1, mode, out, clk);  // warm-up
    CK(hipGetLastError());
    CK(hipDeviceSynchronize());
    CK(hipEventRecord(e0));
    hipLaunchKernelGGL(mfma_loop, dim3(grid), dim3(512), 0, 0, iters, mode, out, clk);
    CK(hipGetLastError());
    CK(hipEventRecord(e1));
    CK(hipEventSynchronize(e1));
    float ms = 0.f;
    CK(hipEventElapsedTime(&ms, e0, e1));
    CK(hipMemcpy(h.data(), clk, h.size() * sizeof(unsigned long long), hipMemcpyDeviceToHost));
    double cyc = 0, real = 0;
    for (long w = 0; w < waves; ++w) cyc += (double)h[2 * w], real += (double)h[2 * w + 1];
    const double ghz = cyc / real * 0.1;  // real-time counter: 100 MHz
    const double flops = (double)waves * iters * 8 * 2.0 * 32 * 32 * 16;
    const double tf = flops / (ms * 1e-3) / 1e12;
    // the dense peak at the measured clock: 1024 SIMDs x 1024 flop per cycle
    // (one 32x32x16 MFMA, 32768 flop, every 32 cycles)
    const double peak_at_clock = 1024.0 * 1024.0 * ghz / 1e3;  // TFLOP/s
    printf("mfma_probe %-6s workgroups %d iters %d: %.3f ms  %.1f TFLOP/s  %.1f%% of 2.5 PFLOP/s  clock %.2f GHz  "
           "%.1f%% of the peak at that clock\n",
           names[mode], grid, iters, ms, tf, tf / 25.0, ghz, 100.0 * tf / peak_at_clock);
  }
  CK(hipFree(out));
  CK(hipFree(clk));
  return 0;
}
