// Multi-head attention for the fp32 DiT path: O = softmax(q k^T / sqrt(dh)) v
// with fp32 products, fp32 exp and fp32 accumulation (online softmax over
// 32-key tiles staged in LDS).  Four lanes share one query, each owning a
// quarter of head_dim; a dot product is reduced over those four lanes.  The
// fp32 path serves the small single-block configuration, which is
// latency-bound, so this kernel favours exactness over matrix-core use.
#include "common.h"
#include "kernels.h"

namespace ditmi {

template <int DH>
__global__ __launch_bounds__(256) void attn_f32_kernel(AttnArgs a) {
  constexpr int SL = DH / 4;  // head_dim slice per lane
  constexpr int BKV = 32;
  __shared__ __attribute__((aligned(16))) float Ks[BKV][DH];
  __shared__ __attribute__((aligned(16))) float Vs[BKV][DH];

  const int tid = threadIdx.x, sub = tid & 3;
  const int b = blockIdx.z, h = blockIdx.y;
  const int Tj = a.Tj;
  const int qi = blockIdx.x * 64 + (tid >> 2);
  const long bh = (long)b * a.H + h;
  const float* __restrict__ qp = (const float*)a.q + bh * Tj * DH;
  const float* __restrict__ kp = (const float*)a.k + bh * Tj * DH;
  const float* __restrict__ vp = (const float*)a.v + bh * Tj * DH;

  float q[SL], o[SL];
#pragma unroll
  for (int d = 0; d < SL; ++d) {
    q[d] = qi < Tj ? qp[(long)qi * DH + sub * SL + d] : 0.f;
    o[d] = 0.f;
  }
  float m_run = -INFINITY, l_run = 0.f;
  for (int kv0 = 0; kv0 < Tj; kv0 += BKV) {
    __syncthreads();
    for (int i = tid; i < BKV * DH; i += 256) {
      const int key = i / DH, d = i - key * DH;
      const bool ok = kv0 + key < Tj;
      Ks[key][d] = ok ? kp[(long)(kv0 + key) * DH + d] : 0.f;
      Vs[key][d] = ok ? vp[(long)(kv0 + key) * DH + d] : 0.f;
    }
    __syncthreads();
    float s[BKV];
    float mt = -INFINITY;
#pragma unroll
    for (int j = 0; j < BKV; ++j) {
      float part = 0.f;
#pragma unroll
      for (int d = 0; d < SL; ++d) part = fmaf(q[d], Ks[j][sub * SL + d], part);
      part += __shfl_xor(part, 1, 64);
      part += __shfl_xor(part, 2, 64);
      s[j] = (kv0 + j < Tj) ? part * a.scale : -INFINITY;
      mt = fmaxf(mt, s[j]);
    }
    const float m_new = fmaxf(m_run, mt);
    const float alpha = expf(m_run - m_new);
    l_run *= alpha;
#pragma unroll
    for (int d = 0; d < SL; ++d) o[d] *= alpha;
#pragma unroll
    for (int j = 0; j < BKV; ++j) {
      const float p = expf(s[j] - m_new);
      l_run += p;
#pragma unroll
      for (int d = 0; d < SL; ++d) o[d] = fmaf(p, Vs[j][sub * SL + d], o[d]);
    }
    m_run = m_new;
  }
  if (qi < Tj) {
    const float inv = 1.0f / l_run;
    const long orow = qi < a.T_img ? (long)b * a.T_img + qi
                                   : (long)a.B * a.T_img + (long)b * a.T_txt + (qi - a.T_img);
    float* op = (float*)a.o + orow * a.D + h * DH + sub * SL;
#pragma unroll
    for (int d = 0; d < SL; ++d) op[d] = o[d] * inv;
  }
}

hipError_t launch_attn_f32(const AttnArgs& a, int head_dim, hipStream_t st) {
  dim3 grid((a.Tj + 63) / 64, a.H, a.B), block(256);
  switch (head_dim) {
    case 64: hipLaunchKernelGGL((attn_f32_kernel<64>), grid, block, 0, st, a); break;
    case 72: hipLaunchKernelGGL((attn_f32_kernel<72>), grid, block, 0, st, a); break;
    case 128: hipLaunchKernelGGL((attn_f32_kernel<128>), grid, block, 0, st, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace ditmi
