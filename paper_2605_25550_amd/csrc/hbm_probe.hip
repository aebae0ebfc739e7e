// Measurement tool (not part of the library): achievable HBM bandwidth on
// one GPU, for comparison with the nominal 8 TB/s.  Two kernels over a
// buffer of MIB mebibytes, 16 bytes per lane per access, grid-stride over
// 256-thread workgroups (8 per CU):
//   copy: dst[i] = src[i]           (bytes moved: 2 x size)
//   read: per-thread sums of src[i], one store per thread (size)
//   hbm_probe [MIB]
// Each is run 3 times untimed, then 20 times between two events.
#include <hip/hip_runtime.h>
#include <cstdio>
#include <cstdlib>

#define CK(x)                                                                            \
  do {                                                                                   \
    hipError_t e_ = (x);                                                                 \
    if (e_ != hipSuccess) {                                                              \
      printf("HIP %s line %d\n", hipGetErrorString(e_), __LINE__);                       \
      exit(1);                                                                           \
    }                                                                                    \
  } while (0)

typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;

__global__ __launch_bounds__(256) void copy_kernel(const f32x4* __restrict__ src, f32x4* __restrict__ dst, long n) {
  const long stride = (long)gridDim.x * blockDim.x;
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) dst[i] = src[i];
}

__global__ __launch_bounds__(256) void read_kernel(const f32x4* __restrict__ src, float* __restrict__ out, long n) {
  const long stride = (long)gridDim.x * blockDim.x;
  const long t = (long)blockIdx.x * blockDim.x + threadIdx.x;
  f32x4 s = {0.f, 0.f, 0.f, 0.f};
  for (long i = t; i < n; i += stride) s += src[i];
  out[t] = (s[0] + s[1]) + (s[2] + s[3]);
}

__global__ void fill_kernel(f32x4* p, long n) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = f32x4{1.f, 2.f, 3.f, 4.f};
}

int main(int argc, char** argv) {
  const long mib = argc > 1 ? atol(argv[1]) : 4096;
  if (mib < 1 || mib > 65536) {
    printf("usage: hbm_probe [MIB 1..65536]\n");
    return 1;
  }
  const long n = mib * (1L << 20) / 16;  // f32x4 elements
  const int grid = 256 * 8;
  f32x4 *a, *b;
  float* out;
  CK(hipMalloc(&a, n * 16));
  CK(hipMalloc(&b, n * 16));
  CK(hipMalloc(&out, (long)grid * 256 * sizeof(float)));
  hipLaunchKernelGGL(fill_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, 0, a, n);
  CK(hipGetLastError());
  CK(hipDeviceSynchronize());
  hipEvent_t e0, e1;
  CK(hipEventCreate(&e0));
  CK(hipEventCreate(&e1));
  for (int k = 0; k < 2; ++k) {
    for (int r = 0; r < 23; ++r) {
      if (r == 3) CK(hipEventRecord(e0));
      if (k == 0) hipLaunchKernelGGL(copy_kernel, dim3(grid), dim3(256), 0, 0, a, b, n);
      else hipLaunchKernelGGL(read_kernel, dim3(grid), dim3(256), 0, 0, a, out, n);
      CK(hipGetLastError());
    }
    CK(hipEventRecord(e1));
    CK(hipEventSynchronize(e1));
    float ms = 0.f;
    CK(hipEventElapsedTime(&ms, e0, e1));
    const double us = ms * 1e3 / 20, bytes = (k == 0 ? 2.0 : 1.0) * n * 16;
    const double gbs = bytes / (us * 1e-6) / 1e9;
    printf("hbm_probe %-4s %ld MiB: %.1f us  %.0f GB/s  %.1f%% of 8 TB/s\n", k == 0 ? "copy" : "read", mib, us, gbs,
           gbs / 80.0);
  }
  CK(hipFree(a));
  CK(hipFree(b));
  CK(hipFree(out));
  return 0;
}
