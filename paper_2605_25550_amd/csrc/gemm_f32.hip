// fp32 GEMM for the fp32 DiT path: y[M, N] = A[M, K] * W[N, K]^T + bias with
// true fp32 products and fp32 accumulation on the vector ALUs (gfx950 has no
// reduced-precision fp32 matrix shortcut, and the fp32 path's tolerance needs
// full fp32 products).  64 x 64 x 16 tiles in LDS (stored k-major so each
// thread reads float4 rows of A and W), 4 x 4 outputs per thread, followed by
// the same fused epilogues as the bf16 GEMM.
#include "common.h"
#include "kernels.h"

namespace ditmi {

template <int EPI>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgs args) {
  constexpr int BM = 64, BN = 64, BK = 16;
  __shared__ __attribute__((aligned(16))) float As[BK][BM + 4];
  __shared__ __attribute__((aligned(16))) float Bs[BK][BN + 4];

  const int tile = blockIdx.x;
  const int pi = (args.nprob > 1 && tile >= args.p[1].tile_begin) ? 1 : 0;
  const GemmProb& P = args.p[pi];
  const int local = tile - P.tile_begin;
  const int m0 = (local / P.tiles_n) * BM, n0 = (local % P.tiles_n) * BN;
  const float* __restrict__ A = (const float*)P.A;
  const float* __restrict__ W = (const float*)P.W;
  const int M = P.M, N = P.N, K = P.K;
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;

  const int lrow = tid >> 2, lk = (tid & 3) * 4;
  const float* a_src = A + (long)min(m0 + lrow, M - 1) * K + lk;
  const float* b_src = W + (long)min(n0 + lrow, N - 1) * K + lk;

  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += BK) {
    float4 av = *(const float4*)(a_src + k0);
    float4 bv = *(const float4*)(b_src + k0);
    __syncthreads();
    As[lk + 0][lrow] = av.x; As[lk + 1][lrow] = av.y; As[lk + 2][lrow] = av.z; As[lk + 3][lrow] = av.w;
    Bs[lk + 0][lrow] = bv.x; Bs[lk + 1][lrow] = bv.y; Bs[lk + 2][lrow] = bv.z; Bs[lk + 3][lrow] = bv.w;
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < BK; ++kk) {
      float4 a4 = *(const float4*)&As[kk][ty * 4];
      float4 b4 = *(const float4*)&Bs[kk][tx * 4];
      float a_[4] = {a4.x, a4.y, a4.z, a4.w}, b_[4] = {b4.x, b4.y, b4.z, b4.w};
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a_[i], b_[j], acc[i][j]);
    }
  }

  const float* __restrict__ bias = (const float*)P.bias;
  const int rpb = P.rows_per_batch;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty * 4 + i;
    if (m >= M) continue;
    const int b = m / rpb;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + tx * 4 + j;
      if (n >= N) continue;
      const float y = acc[i][j] + bias[n];
      if (EPI == EPI_RESID || EPI == EPI_RESID2) {
        float* xr = P.resid + (long)m * N + n;
        *xr = *xr + P.gate[(long)b * P.gate_stride + n] * y;
      } else if (EPI == EPI_GELU) {
        ((float*)P.out)[(long)m * N + n] = gelu_tanh(y);
      } else if (EPI == EPI_STORE) {
        ((float*)P.out)[(long)m * N + n] = y;
      } else {
        const int s = n / P.hidden, rem = n - s * P.hidden;
        const int h = rem / P.head_dim, d = rem - h * P.head_dim;
        const int jpos = m - b * rpb + P.seq_off;
        float* dst = (float*)(s == 0 ? P.q : (s == 1 ? P.k : P.v));
        const int stride = s == 2 ? P.head_dim : P.qk_stride;
        dst[(((long)b * P.heads + h) * P.Tj + jpos) * stride + d] = y;
      }
    }
  }
}

hipError_t launch_gemm_f32(const GemmArgs& a, int epi, hipStream_t st) {
  dim3 grid(a.total_tiles), block(256);
  switch (epi) {
    case EPI_QKV: hipLaunchKernelGGL((gemm_f32_kernel<EPI_QKV>), grid, block, 0, st, a); break;
    case EPI_GELU: hipLaunchKernelGGL((gemm_f32_kernel<EPI_GELU>), grid, block, 0, st, a); break;
    case EPI_RESID: hipLaunchKernelGGL((gemm_f32_kernel<EPI_RESID>), grid, block, 0, st, a); break;
    case EPI_RESID2: hipLaunchKernelGGL((gemm_f32_kernel<EPI_RESID2>), grid, block, 0, st, a); break;
    default: hipLaunchKernelGGL((gemm_f32_kernel<EPI_STORE>), grid, block, 0, st, a); break;
  }
  return hipGetLastError();
}

}  // namespace ditmi
