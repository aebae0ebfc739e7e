// Measurement tool (not part of the library): times the bf16 GEMM kernels
// of the library in isolation for given shapes and tile configurations, to
// compare tile choices on one GPU.
//   gemm_probe "M N K epi tile split [group_m]" ...
// epi: 1 GELU (bf16 out), 2 / 4 residual (fp32); tile: kernels.h TILE_*;
// split: k-ranges of the problem (0 = none); group_m: tile-order group
// height (default 8).  Operands are pseudo-random bf16; every case is run 5
// times untimed, then 30 times between two events.  Prints us per launch,
// TFLOP/s and % of 2.5 PFLOP/s.
#include <hip/hip_runtime.h>
#include <cstdio>
#include <cstdlib>
#include <vector>
#include "kernels.h"
using namespace ditmi;
#define CK(x) do { hipError_t e_ = (x); if (e_ != hipSuccess) { printf("HIP %s line %d\n", hipGetErrorString(e_), __LINE__); exit(1);} } while (0)
__global__ void fill_bf16(uint16_t* p, long n, unsigned seed) {
  long i = blockIdx.x * 256L + threadIdx.x;
  if (i >= n) return;
  unsigned h = (unsigned)i * 2654435761u ^ seed; h ^= h >> 15; h *= 2246822519u; h ^= h >> 13;
  float z = ((h & 0xFFFF) / 65536.0f - 0.5f) * 0.1f;
  p[i] = (uint16_t)(__float_as_uint(z) >> 16);
}
__global__ void fill_f32(float* p, long n, float v) { long i = blockIdx.x * 256L + threadIdx.x; if (i < n) p[i] = v; }
int main(int argc, char** argv) {
  long maxA = 0, maxW = 0, maxC = 0;
  struct Case { int M, N, K, epi, tile, split, gm; };  // (EPI_QKV and EPI_STORE are not probed)
  std::vector<Case> cs;
  for (int i = 1; i < argc; ++i) { Case c; c.gm = 8; sscanf(argv[i], "%d %d %d %d %d %d %d", &c.M, &c.N, &c.K, &c.epi, &c.tile, &c.split, &c.gm); cs.push_back(c);
    maxA = std::max(maxA, (long)c.M * c.K); maxW = std::max(maxW, (long)c.N * c.K); maxC = std::max(maxC, (long)c.M * c.N); }
  uint16_t *A, *W, *bias, *out; float *resid, *gate, *part;
  CK(hipMalloc(&A, maxA * 2)); CK(hipMalloc(&W, maxW * 2)); CK(hipMalloc(&bias, 65536 * 2));
  CK(hipMalloc(&out, maxC * 2)); CK(hipMalloc(&resid, maxC * 4)); CK(hipMalloc(&gate, 65536 * 4));
  CK(hipMalloc(&part, maxC * 4 * 8));
  fill_bf16<<<(maxA + 255) / 256, 256>>>(A, maxA, 1); fill_bf16<<<(maxW + 255) / 256, 256>>>(W, maxW, 2);
  fill_bf16<<<256, 256>>>(bias, 65536, 3); fill_f32<<<(maxC + 255) / 256, 256>>>(resid, maxC, 0.f);
  fill_f32<<<256, 256>>>(gate, 65536, 0.5f);
  CK(hipDeviceSynchronize());
  hipEvent_t e0, e1; CK(hipEventCreate(&e0)); CK(hipEventCreate(&e1));
  for (auto& c : cs) {
    GemmArgs a{}; a.nprob = 1;
    GemmProb& p = a.p[0];
    p.A = A; p.W = W; p.bias = bias; p.M = c.M; p.N = c.N; p.K = c.K; p.rows_per_batch = c.M;
    p.resid = resid; p.gate = gate; p.gate_stride = 0; p.out = out;
    int bm, bn; gemm_tile_dims(c.tile, &bm, &bn);
    p.tiles_m = (c.M + bm - 1) / bm; p.tiles_n = (c.N + bn - 1) / bn; p.tile_begin = 0; p.group_m = c.gm;
    a.total_tiles = p.tiles_m * p.tiles_n;
    if (c.split > 1) { p.ksplit = c.split; p.part = part; a.total_tiles *= c.split; }
    for (int w = 0; w < 5; ++w) CK(launch_gemm_bf16(a, c.epi, c.tile, 0));
    CK(hipDeviceSynchronize());
    const int R = 30;
    CK(hipEventRecord(e0, 0));
    for (int r = 0; r < R; ++r) CK(launch_gemm_bf16(a, c.epi, c.tile, 0));
    CK(hipEventRecord(e1, 0)); CK(hipEventSynchronize(e1));
    float ms; CK(hipEventElapsedTime(&ms, e0, e1));
    double us = ms * 1e3 / R, tf = 2.0 * c.M * c.N * c.K / (us * 1e-6) / 1e12;
    printf("M %d N %d K %d epi %d tile %d (%dx%d) split %d gm %d tiles %d: %.2f us  %.1f TFLOP/s  %.1f%%\n", c.M, c.N, c.K, c.epi, c.tile, bm, bn, c.split, c.gm, a.total_tiles, us, tf, tf / 25.0);
    fflush(stdout);
  }
  return 0;
}
