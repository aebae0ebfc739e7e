// Memory-bound kernels of the DiT step on gfx950:
//   * LayerNorm + adaLN modulate: h = LN(x) * (1 + scale) + shift, fp32 in,
//     GEMM operand (bf16 or fp32) out; one wavefront per token row, 16-byte
//     loads, exact two-pass mean/variance from registers.
//   * adaLN modulation GEMV: m = SiLU(c) W_ada^T + b_ada for many (block,
//     stream) weight matrices in one launch; HBM-bound on the weights.
//   * timestep + class conditioning, patch embedding, 2-D sin-cos table.
#include <math.h>

#include "common.h"
#include "kernels.h"

namespace ditmi {

// ---------------------------------------------------------------- LayerNorm + modulate
template <typename OutT, int NV>
__global__ __launch_bounds__(256) void ln_mod_kernel(LnArgs a) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= a.total_rows) return;  // whole wavefront leaves together
  const int si = (a.nseg > 1 && row >= a.s[1].row_begin) ? 1 : 0;
  // select by value: indexing the by-value argument array with a runtime
  // index would copy it to scratch memory
  const LnSeg S = si ? a.s[1] : a.s[0];
  const int r = row - S.row_begin;
  const int b = r / S.rows_per_batch;
  const int D = a.D, nq = D >> 2;
  const f32x4* __restrict__ xr = (const f32x4*)(S.x + (long)r * D);

  // shift/scale are loaded with x, before the reductions, so that their
  // latency overlaps the row's.  Loads use a clamped (always valid) index and
  // the values are selected afterwards; vectors are clang ext_vector types
  // (HIP's float4/uint2 structs, kept in arrays, are placed in memory).
  const f32x4* __restrict__ sh = (const f32x4*)(S.shift + (long)b * S.mod_stride);
  const f32x4* __restrict__ sc = (const f32x4*)(S.scale + (long)b * S.mod_stride);
  f32x4 v[NV], s4[NV], c4[NV];
  float sum = 0.f;
  const f32x4 z = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int c = lane + 64 * i;
    const int cc = min(c, nq - 1);
    const bool in = c < nq;
    const f32x4 tx = xr[cc], ts = sh[cc], tc = sc[cc];
    v[i] = in ? tx : z;
    s4[i] = in ? ts : z;
    c4[i] = in ? tc : z;
    sum += (v[i][0] + v[i][1]) + (v[i][2] + v[i][3]);
  }
  const float mean = wave_sum(sum) / (float)D;
  float sq = 0.f;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int c = lane + 64 * i;
    const f32x4 d = v[i] - mean;
    const float q = (d[0] * d[0] + d[1] * d[1]) + (d[2] * d[2] + d[3] * d[3]);
    sq += c < nq ? q : 0.f;
  }
  const float var = wave_sum(sq) / (float)D;
  const float rstd = 1.0f / sqrtf(var + a.eps);
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int c = lane + 64 * i;
    if (c >= nq) continue;
    const f32x4 y = (v[i] - mean) * rstd * (1.f + c4[i]) + s4[i];
    if constexpr (sizeof(OutT) == 2) {
      ((u32x2*)S.out)[(long)r * nq + c] = u32x2{pack_bf16x2(y[0], y[1]), pack_bf16x2(y[2], y[3])};
    } else {
      ((f32x4*)S.out)[(long)r * nq + c] = y;
    }
  }
}

template <typename OutT>
static hipError_t ln_dispatch(const LnArgs& a, hipStream_t st) {
  dim3 grid((a.total_rows + 3) / 4), block(256);
  const int nv = (a.D / 4 + 63) / 64;
  if (nv <= 2) hipLaunchKernelGGL((ln_mod_kernel<OutT, 2>), grid, block, 0, st, a);
  else if (nv <= 5) hipLaunchKernelGGL((ln_mod_kernel<OutT, 5>), grid, block, 0, st, a);
  else if (nv <= 8) hipLaunchKernelGGL((ln_mod_kernel<OutT, 8>), grid, block, 0, st, a);
  else if (nv <= 12) hipLaunchKernelGGL((ln_mod_kernel<OutT, 12>), grid, block, 0, st, a);
  else hipLaunchKernelGGL((ln_mod_kernel<OutT, 16>), grid, block, 0, st, a);
  return hipGetLastError();
}

hipError_t launch_ln_mod(const LnArgs& a, int dtype, hipStream_t st) {
  return dtype == 1 ? ln_dispatch<bf16_t>(a, st) : ln_dispatch<float>(a, st);
}

// ---------------------------------------------------------------- adaLN GEMV
// Workgroup = 4 waves x 8 lane-groups x 4 rows = 128 output rows of one
// entry.  A lane-group of 8 lanes reads 128 contiguous bytes of each of its
// 4 weight rows per step; SiLU(c) for up to 8 samples sits in LDS and is
// reused across the 4 rows.
template <typename WT> struct W8;
template <> struct W8<bf16_t> {
  static __device__ __forceinline__ void load(const bf16_t* p, float* w) {
    uint4 u = *(const uint4*)p;
    uint32_t x[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      w[2 * i] = __uint_as_float(x[i] << 16);
      w[2 * i + 1] = __uint_as_float(x[i] & 0xFFFF0000u);
    }
  }
};
template <> struct W8<float> {
  static __device__ __forceinline__ void load(const float* p, float* w) {
    float4 u0 = *(const float4*)p, u1 = *(const float4*)(p + 4);
    w[0] = u0.x; w[1] = u0.y; w[2] = u0.z; w[3] = u0.w;
    w[4] = u1.x; w[5] = u1.y; w[6] = u1.z; w[7] = u1.w;
  }
};

template <typename WT>
__global__ __launch_bounds__(256) void adaln_kernel(AdaArgs a) {
  extern __shared__ float sc[];  // [min(B, 8)][D]
  const int wg = blockIdx.x;
  int ei = 0;
  while (ei + 1 < a.ne && wg >= a.e[ei + 1].wg_begin) ++ei;
  const AdaEntry& E = a.e[ei];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int grp = lane >> 3, li = lane & 7;
  const int nbase = (wg - E.wg_begin) * 128 + wave * 32 + grp * 4;
  const WT* __restrict__ W = (const WT*)E.W;
  const WT* __restrict__ bias = (const WT*)E.bias;
  const int D = a.D, nch = D >> 3, N = E.N;

  for (int b0 = 0; b0 < a.B; b0 += 8) {
    const int nb = min(8, a.B - b0);
    __syncthreads();
    for (int i = tid; i < nb * D; i += 256) {
      const float z = a.cond[(long)b0 * D + i];
      sc[i] = z / (1.0f + expf(-z));
    }
    __syncthreads();
    float acc[4][8];
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int bb = 0; bb < 8; ++bb) acc[r][bb] = 0.f;
    for (int ci = li; ci < nch; ci += 8) {
      float w[4][8];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int n = nbase + r;
        if (n < N) W8<WT>::load(W + (long)n * D + ci * 8, w[r]);
        else
#pragma unroll
          for (int e = 0; e < 8; ++e) w[r][e] = 0.f;
      }
#pragma unroll
      for (int bb = 0; bb < 8; ++bb) {
        if (bb < nb) {
          const float4 s0 = *(const float4*)&sc[bb * D + ci * 8];
          const float4 s1 = *(const float4*)&sc[bb * D + ci * 8 + 4];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            float t = acc[r][bb];
            t = fmaf(w[r][0], s0.x, t); t = fmaf(w[r][1], s0.y, t);
            t = fmaf(w[r][2], s0.z, t); t = fmaf(w[r][3], s0.w, t);
            t = fmaf(w[r][4], s1.x, t); t = fmaf(w[r][5], s1.y, t);
            t = fmaf(w[r][6], s1.z, t); t = fmaf(w[r][7], s1.w, t);
            acc[r][bb] = t;
          }
        }
      }
    }
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int bb = 0; bb < 8; ++bb) {
        float t = acc[r][bb];
        t += __shfl_xor(t, 1, 64);
        t += __shfl_xor(t, 2, 64);
        t += __shfl_xor(t, 4, 64);
        acc[r][bb] = t;
      }
    // lane li of the group writes sample b0 + li
    if (li < nb) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int n = nbase + r;
        if (n >= N) continue;
        float val = 0.f;
#pragma unroll
        for (int bb = 0; bb < 8; ++bb) val = (bb == li) ? acc[r][bb] : val;
        E.out[(long)(b0 + li) * N + n] = val + ld_as_float<WT>(bias, n);
      }
    }
  }
}

// bf16 weights: the same product on v_mfma_f32_16x16x32_bf16 as
// out^T [N, B] = W [N, K] * SiLU(c)^T [K, B].  A workgroup (4 waves x 4 row
// tiles of 16) owns 256 rows of one entry; each B fragment feeds the four
// row tiles.  Both operands are read straight from global memory, 16 bytes
// per lane (row lane%16, k offset 8*(lane/16)): W streams from HBM once,
// and the B operand, SiLU(c) in bf16 for 16 samples (computed once by
// silu_bf16_kernel, zero rows past the batch; at most a few hundred KB),
// stays in L2; lanes of samples past the batch supply zeros without a load
// (at batch 1, fifteen of sixteen).  No LDS, so many workgroups share a CU
// and keep enough weight loads in flight to stream HBM (staging the B
// operand in LDS held one workgroup per CU at hidden 3072).  Measured:
// 4.2 TB/s with two row tiles per wave and every lane loading, 4.7-5.2 TB/s
// like this (a plain streaming read of the same rows: 5.8-6.1).  Batches
// above 16 loop over 16-sample tiles.  D lanes hold column (sample)
// lane%16, rows 4*(lane/16) + i.
__global__ void silu_bf16_kernel(int B, int D, int rows, const float* cond, bf16_t* act) {
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long)rows * D) return;
  const int r = (int)(idx / D);
  act[idx] = r < B ? f2bf(silu(cond[idx])) : (bf16_t)0;
}

hipError_t launch_silu_bf16(int B, int D, const float* cond, void* act, hipStream_t st) {
  const int rows = (B + 15) / 16 * 16;
  const long n = (long)rows * D;
  hipLaunchKernelGGL(silu_bf16_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, B, D, rows, cond,
                     (bf16_t*)act);
  return hipGetLastError();
}

__global__ __launch_bounds__(256) void adaln_mfma_kernel(AdaArgs a) {
  constexpr int RT = ADA_ROWS_PER_WG / 64;  // row tiles of 16 per wave
  const int wg = blockIdx.x;
  int ei = 0;
  while (ei + 1 < a.ne && wg >= a.e[ei + 1].wg_begin) ++ei;
  const AdaEntry& E = a.e[ei];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int K = a.D, N = E.N;
  const int nbase = (wg - E.wg_begin) * ADA_ROWS_PER_WG + wave * (16 * RT);
  const bf16_t* __restrict__ W = (const bf16_t*)E.W;
  const bf16_t* __restrict__ bias = (const bf16_t*)E.bias;
  const bf16_t* __restrict__ act = (const bf16_t*)a.act;
  const int r16 = lane & 15, kq = lane >> 4;
  const bf16_t* wr[RT];
#pragma unroll
  for (int t = 0; t < RT; ++t) wr[t] = W + (long)min(nbase + 16 * t + r16, N - 1) * K + 8 * kq;

  for (int b0 = 0; b0 < a.B; b0 += 16) {
    const bool live = b0 + r16 < a.B;  // this lane's sample exists
    const bf16_t* sp = act + (long)(b0 + r16) * K + 8 * kq;
    f32x4 acc[RT];
#pragma unroll
    for (int t = 0; t < RT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll 8
    for (int k0 = 0; k0 < K; k0 += 32) {
      const bf16x8 bv = live ? *(const bf16x8*)(sp + k0) : bf16x8{};
#pragma unroll
      for (int t = 0; t < RT; ++t)
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(*(const bf16x8*)(wr[t] + k0), bv, acc[t], 0, 0, 0);
    }
    const int b = b0 + r16;
    if (b < a.B) {
#pragma unroll
      for (int t = 0; t < RT; ++t) {
        const int n = nbase + 16 * t + 4 * kq;  // N is a multiple of 4
        if (n >= N) continue;
        const f32x4 v = acc[t];
        *(f32x4*)(E.out + (long)b * N + n) =
            f32x4{v[0] + bf2f(bias[n]), v[1] + bf2f(bias[n + 1]), v[2] + bf2f(bias[n + 2]), v[3] + bf2f(bias[n + 3])};
      }
    }
  }
}

hipError_t launch_adaln(const AdaArgs& a, int dtype, hipStream_t st) {
  dim3 grid(a.total_wg), block(256);
  if (dtype == 1) {
    hipLaunchKernelGGL(adaln_mfma_kernel, grid, block, 0, st, a);
  } else {
    const size_t lds = (size_t)(a.B < 8 ? a.B : 8) * a.D * sizeof(float);
    hipError_t e = hipFuncSetAttribute((const void*)adaln_kernel<float>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((adaln_kernel<float>), grid, block, lds, st, a);
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------- conditioning
// feat[b][i] = cos(t_b f_i) (i < 128), sin(t_b f_{i-128}) (i >= 128),
// f_i = exp(-ln(10000) i / 128); evaluated in double for the large arguments.
__global__ void timestep_feat_kernel(int B, const float* t, float* feat) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= B * 256) return;
  const int b = idx >> 8, i = idx & 255;
  const int fi = i & 127;
  const double f = exp(-9.210340371976184 * (double)fi / 128.0);  // ln(10000)
  const double arg = (double)t[b] * f;
  feat[idx] = (float)(i < 128 ? cos(arg) : sin(arg));
}

// out[b][n] = post(sum_k W[n][k] in[b][k] + bias[n]); one wavefront per row n.
// The row is loaded once into registers (8 consecutive weights per lane and
// chunk, 16-byte loads) and dotted with every sample's input vector.
// MODE 0: post = SiLU.  MODE 1: post = identity, plus class_table[y[b]][n].
// K is a multiple of 8 and at most 8 * 64 * RD_MAXCH.
constexpr int RD_MAXCH = 8;
template <typename WT, int MODE>
__global__ __launch_bounds__(256) void rowdot_kernel(int B, int N, int K, const float* in, const WT* W,
                                                     const WT* bias, const WT* table, const int32_t* y,
                                                     float* out) {
  const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (n >= N) return;
  const int nch = K >> 3;
  float w[RD_MAXCH][8];
#pragma unroll
  for (int i = 0; i < RD_MAXCH; ++i) {
    const int c = lane + 64 * i;
    if (c < nch) W8<WT>::load(W + (long)n * K + c * 8, w[i]);
    else
#pragma unroll
      for (int e = 0; e < 8; ++e) w[i][e] = 0.f;
  }
  const float bn = ld_as_float<WT>(bias, n);
  for (int b = 0; b < B; ++b) {
    const float* xb = in + (long)b * K;
    float acc = 0.f;
#pragma unroll
    for (int i = 0; i < RD_MAXCH; ++i) {
      const int c = lane + 64 * i;
      if (c < nch) {
        const float4 x0 = *(const float4*)(xb + c * 8), x1 = *(const float4*)(xb + c * 8 + 4);
        acc = fmaf(w[i][0], x0.x, acc); acc = fmaf(w[i][1], x0.y, acc);
        acc = fmaf(w[i][2], x0.z, acc); acc = fmaf(w[i][3], x0.w, acc);
        acc = fmaf(w[i][4], x1.x, acc); acc = fmaf(w[i][5], x1.y, acc);
        acc = fmaf(w[i][6], x1.z, acc); acc = fmaf(w[i][7], x1.w, acc);
      }
    }
    acc = wave_sum(acc) + bn;
    if (lane == 0) {
      if (MODE == 0) out[(long)b * N + n] = acc / (1.0f + expf(-acc));
      else out[(long)b * N + n] = acc + ld_as_float<WT>(table, (long)y[b] * N + n);
    }
  }
}

hipError_t launch_cond_embed(int B, int D, const float* t, const int32_t* y, const void* w1, const void* b1,
                             const void* w2, const void* b2, const void* table, float* feat, float* h1,
                             float* cond, int dtype, hipStream_t st) {
  hipLaunchKernelGGL(timestep_feat_kernel, dim3((B * 256 + 255) / 256), dim3(256), 0, st, B, t, feat);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  dim3 grid((D + 3) / 4), block(256);
  if (dtype == 1) {
    hipLaunchKernelGGL((rowdot_kernel<bf16_t, 0>), grid, block, 0, st, B, D, 256, feat, (const bf16_t*)w1,
                       (const bf16_t*)b1, (const bf16_t*)nullptr, (const int32_t*)nullptr, h1);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL((rowdot_kernel<bf16_t, 1>), grid, block, 0, st, B, D, D, h1, (const bf16_t*)w2,
                       (const bf16_t*)b2, (const bf16_t*)table, y, cond);
  } else {
    hipLaunchKernelGGL((rowdot_kernel<float, 0>), grid, block, 0, st, B, D, 256, feat, (const float*)w1,
                       (const float*)b1, (const float*)nullptr, (const int32_t*)nullptr, h1);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL((rowdot_kernel<float, 1>), grid, block, 0, st, B, D, D, h1, (const float*)w2,
                       (const float*)b2, (const float*)table, y, cond);
  }
  return hipGetLastError();
}

// Patch embedding x = z W^T + b (+ pos), fp32 accumulation in the order
// b, p = 0 .. P-1, then pos.
//
// Up to 16 channels (patch_row_kernel): one workgroup per token row, the
// patch vector in LDS, each lane a column.
template <typename WT>
__global__ __launch_bounds__(256) void patch_row_kernel(int T, int P, int D, const float* __restrict__ z,
                                                        const WT* __restrict__ w, const WT* __restrict__ bias,
                                                        const float* __restrict__ pos, float* __restrict__ x) {
  __shared__ float zs[16];
  const int row = blockIdx.x, tid = threadIdx.x;
  if (tid < P) zs[tid] = z[(long)row * P + tid];
  __syncthreads();
  const int t = row % T;
  for (int n = tid; n < D; n += 256) {
    float acc = ld_as_float<WT>(bias, n);
    const WT* wr = w + (long)n * P;
    for (int p = 0; p < P; ++p) acc = fmaf(ld_as_float<WT>(wr, p), zs[p], acc);
    if (pos) acc += pos[(long)t * D + n];
    x[(long)row * D + n] = acc;
  }
}

// More channels (patch_tile_kernel): a workgroup owns 256 consecutive
// columns and PT_ROWS rows.  Per chunk of 64 channels, the rows' latent
// values are staged in LDS (read back as one broadcast 16-byte read per four
// channels) and each lane holds its column's 64 weights in registers, so
// every weight element is read once per workgroup instead of once per row.
constexpr int PT_ROWS = 32, PT_CHUNK = 64;

template <typename WT>
__global__ __launch_bounds__(256) void patch_tile_kernel(int rows, int T, int P, int D, const float* __restrict__ z,
                                                         const WT* __restrict__ w, const WT* __restrict__ bias,
                                                         const float* __restrict__ pos, float* __restrict__ x) {
  __shared__ __attribute__((aligned(16))) float zs[PT_ROWS][PT_CHUNK];
  const int tid = threadIdx.x;
  const int n = blockIdx.x * 256 + tid;
  const int r0 = blockIdx.y * PT_ROWS;
  const int nr = min(PT_ROWS, rows - r0);
  const bool col = n < D;
  const float b = col ? ld_as_float<WT>(bias, n) : 0.f;
  float acc[PT_ROWS];
#pragma unroll
  for (int r = 0; r < PT_ROWS; ++r) acc[r] = b;
  for (int p0 = 0; p0 < P; p0 += PT_CHUNK) {
    const int pc = min(PT_CHUNK, P - p0);
    __syncthreads();  // the previous chunk's reads are done
    for (int e = tid; e < PT_ROWS * PT_CHUNK; e += 256) {
      const int r = e / PT_CHUNK, c = e % PT_CHUNK;
      zs[r][c] = r < nr && c < pc ? z[(long)(r0 + r) * P + p0 + c] : 0.f;
    }
    float wv[PT_CHUNK];
    if (col && pc == PT_CHUNK && P % 8 == 0) {
      // the lane's 64 weights as 16-byte loads (8 elements each, aligned:
      // n P + p0 + c is a multiple of 8)
#pragma unroll
      for (int c = 0; c < PT_CHUNK; c += 8) W8<WT>::load(w + (long)n * P + p0 + c, &wv[c]);
    } else {
#pragma unroll
      for (int c = 0; c < PT_CHUNK; ++c) wv[c] = col && c < pc ? ld_as_float<WT>(w, (long)n * P + p0 + c) : 0.f;
    }
    __syncthreads();
    if (pc == PT_CHUNK) {
#pragma unroll
      for (int r = 0; r < PT_ROWS; ++r)
#pragma unroll
        for (int c = 0; c < PT_CHUNK; c += 4) {
          const f32x4 zv = *(const f32x4*)&zs[r][c];
          acc[r] = fmaf(wv[c], zv[0], acc[r]);
          acc[r] = fmaf(wv[c + 1], zv[1], acc[r]);
          acc[r] = fmaf(wv[c + 2], zv[2], acc[r]);
          acc[r] = fmaf(wv[c + 3], zv[3], acc[r]);
        }
    } else {  // last, partial chunk (static register indices, channels c < pc only)
#pragma unroll
      for (int r = 0; r < PT_ROWS; ++r)
#pragma unroll
        for (int c = 0; c < PT_CHUNK; ++c)
          if (c < pc) acc[r] = fmaf(wv[c], zs[r][c], acc[r]);
    }
  }
  if (!col) return;
#pragma unroll
  for (int r = 0; r < PT_ROWS; ++r) {
    if (r >= nr) break;
    const int row = r0 + r;
    float v = acc[r];
    if (pos) v += pos[(long)(row % T) * D + n];
    x[(long)row * D + n] = v;
  }
}

template <typename WT>
static void launch_patch_embed_t(int rows, int T, int P, int D, const float* z, const WT* w, const WT* b,
                                 const float* pos, float* x, hipStream_t st) {
  if (P <= 16)
    hipLaunchKernelGGL((patch_row_kernel<WT>), dim3(rows), dim3(256), 0, st, T, P, D, z, w, b, pos, x);
  else
    hipLaunchKernelGGL((patch_tile_kernel<WT>), dim3((D + 255) / 256, (rows + PT_ROWS - 1) / PT_ROWS), dim3(256), 0,
                       st, rows, T, P, D, z, w, b, pos, x);
}

hipError_t launch_patch_embed(int rows, int T, int P, int D, const float* z, const void* w, const void* b,
                              const float* pos, float* x, int dtype, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  if (dtype == 1)
    launch_patch_embed_t<bf16_t>(rows, T, P, D, z, (const bf16_t*)w, (const bf16_t*)b, pos, x, st);
  else
    launch_patch_embed_t<float>(rows, T, P, D, z, (const float*)w, (const float*)b, pos, x, st);
  return hipGetLastError();
}

// ---------------------------------------------------------------- 2-D sin-cos table
__global__ void pos_embed_2d_kernel(int gh, int gw, int D, float* pos) {
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  const long total = (long)gh * gw * D;
  if (idx >= total) return;
  const int n = (int)(idx / D), dd = (int)(idx - (long)n * D);
  const int r = n / gw, c = n - r * gw;
  const int half = D / 2, q = D / 4;
  const int p = dd < half ? c : r;
  const int e = dd < half ? dd : dd - half;
  const int i = e < q ? e : e - q;
  const double omega = exp(-9.210340371976184 * (double)i / (double)q);  // 10000^(-i/q)
  const double arg = (double)p * omega;
  pos[idx] = (float)(e < q ? sin(arg) : cos(arg));
}

hipError_t launch_pos_embed_2d(int gh, int gw, int D, float* pos, hipStream_t st) {
  const long total = (long)gh * gw * D;
  hipLaunchKernelGGL(pos_embed_2d_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st, gh, gw, D, pos);
  return hipGetLastError();
}

// ---------------------------------------------------------------- sampler loop
// p[i] = v for i < n (per-step timestep for the conditioning; a kernel, not a
// memset, so that the loop can be captured into a HIP graph).
__global__ void fill_f32_kernel(float* p, int n, float v) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

hipError_t launch_fill_f32(float* p, int n, float v, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_f32_kernel, dim3((n + 255) / 256), dim3(256), 0, st, p, n, v);
  return hipGetLastError();
}

// Euler update z += a * v over n floats (n a multiple of 4, 16-byte aligned).
__global__ void axpy_f32_kernel(f32x4* z, const f32x4* v, float a, long n4) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n4) z[i] += a * v[i];
}

hipError_t launch_axpy_f32(float* z, const float* v, float a, long n, hipStream_t st) {
  const long n4 = n / 4;
  if (n4 <= 0) return hipSuccess;
  hipLaunchKernelGGL(axpy_f32_kernel, dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, st, (f32x4*)z,
                     (const f32x4*)v, a, n4);
  return hipGetLastError();
}


}  // namespace ditmi
