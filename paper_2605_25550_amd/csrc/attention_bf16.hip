// Fused multi-head attention, bf16 operands, fp32 softmax and accumulation,
// for gfx950: O = softmax(q k^T / sqrt(dh)) v per (sample, head), the
// O(T^2 D) part of the DiT block.  Flash-style single pass with an online
// softmax, so no T x T score matrix ever reaches HBM.
//
// Orientation.  Each wavefront owns 32 queries.  It computes S^T = K Q^T with
// v_mfma_f32_32x32x16_bf16 (A = a K tile from LDS, B = the wave's Q^T held in
// registers for the whole pass), so every lane holds the scores of ONE query
// (its lane index mod 32) for 32 keys: the row max and row sum are in-lane,
// plus one exchange with the other half-wavefront.  The probabilities are
// then already laid out as the B operand of O^T = V^T P^T (keys permuted
// consistently on both operands), and O^T's accumulators again belong to the
// lane's own query, so the online-softmax rescale is a per-lane scalar.
// V is consumed transposed (v^T [dh][T], written that way by the QKV GEMM
// epilogue) so its A operand is two 8-byte LDS reads per lane.
//
// Tiles: 128 queries per workgroup (4 waves), 64 keys per step, K and V^T
// double-buffered in LDS (global -> VGPR -> LDS; the next tile's loads are in
// flight during the current tile's math).  head_dim 72 is zero-padded to 80
// for the QK^T contraction and to 96 rows of V^T; the last key tile is masked.
#include "common.h"
#include "kernels.h"

namespace ditmi {

template <int DH>
__global__ __launch_bounds__(256) void attn_bf16_kernel(AttnArgs a) {
  constexpr int DHP = (DH + 15) / 16 * 16;  // QK^T contraction length
  constexpr int DT = (DH + 31) / 32;        // 32-row tiles of V^T / O^T
  constexpr int BKV = 64;
  constexpr int KST = DHP + 8;              // LDS row stride of K (bf16)
  constexpr int VST = BKV + 8;              // LDS row stride of V^T (bf16)
  constexpr int KCH = DHP / 8;              // 16-byte chunks per K row
  constexpr int K_IT = (BKV * KCH + 255) / 256;
  constexpr int V_IT = (DH * 8 + 255) / 256;
  __shared__ __attribute__((aligned(16))) bf16_t Ks[2][BKV * KST];
  __shared__ __attribute__((aligned(16))) bf16_t Vs[2][DT * 32 * VST];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 5, r32 = lane & 31;
  const int b = blockIdx.z, h = blockIdx.y;
  const int Tj = a.Tj, Tjp = a.Tj_pad;
  const int qrow = blockIdx.x * 128 + wave * 32 + r32;
  const long bh = (long)b * a.H + h;
  const bf16_t* __restrict__ qp = (const bf16_t*)a.q + bh * Tj * DH;
  const bf16_t* __restrict__ kp = (const bf16_t*)a.k + bh * Tj * DH;
  const bf16_t* __restrict__ vp = (const bf16_t*)a.v + bh * DH * (long)Tjp;

  // V^T rows beyond head_dim only feed discarded O^T rows; keep them finite.
  if (DT * 32 > DH) {
    for (int i = tid; i < (DT * 32 - DH) * VST; i += 256) {
      Vs[0][DH * VST + i] = 0;
      Vs[1][DH * VST + i] = 0;
    }
  }

  bf16x8 qf[DHP / 16];
#pragma unroll
  for (int s = 0; s < DHP / 16; ++s) {
    const int d0 = s * 16 + g * 8;
    if (qrow < Tj && d0 < DH)
      qf[s] = *(const bf16x8*)(qp + (long)qrow * DH + d0);
    else
      qf[s] = bf16x8{};
  }

  u32x4 rk[K_IT], rv[V_IT];
  // Fetch one K / V^T tile (keys kv0 .. kv0+63) into registers; keys past the
  // end and head_dim padding read as zero.
#define ATT_GLOAD(kv0_)                                                                 \
  do {                                                                                 \
    const int kvb = (kv0_);                                                            \
    _Pragma("unroll") for (int i = 0; i < K_IT; ++i) {                                 \
      const int c = tid + 256 * i;                                                     \
      const int key = c / KCH, dc = c - key * KCH;                                     \
      rk[i] = u32x4{0u, 0u, 0u, 0u};                                                   \
      if (c < BKV * KCH && kvb + key < Tj && dc * 8 < DH)                              \
        rk[i] = *(const u32x4*)(kp + (long)(kvb + key) * DH + dc * 8);                 \
    }                                                                                  \
    _Pragma("unroll") for (int i = 0; i < V_IT; ++i) {                                 \
      const int c = tid + 256 * i;                                                     \
      const int d = c >> 3, key0 = kvb + (c & 7) * 8;                                  \
      rv[i] = u32x4{0u, 0u, 0u, 0u};                                                   \
      if (c < DH * 8 && key0 < Tj) {                                                   \
        u32x4 v = *(const u32x4*)(vp + (long)d * Tjp + key0);                          \
        const int nv = Tj - key0;                                                      \
        if (nv < 8) {                                                                  \
          _Pragma("unroll") for (int e = 0; e < 4; ++e) {                              \
            if (2 * e >= nv) v[e] = 0u;                                                \
            else if (2 * e + 1 >= nv) v[e] &= 0xFFFFu;                                 \
          }                                                                            \
        }                                                                              \
        rv[i] = v;                                                                     \
      }                                                                                \
    }                                                                                  \
  } while (0)
#define ATT_LSTORE(buf_)                                                                \
  do {                                                                                 \
    _Pragma("unroll") for (int i = 0; i < K_IT; ++i) {                                 \
      const int c = tid + 256 * i;                                                     \
      if (c < BKV * KCH) {                                                             \
        const int key = c / KCH, dc = c - key * KCH;                                   \
        *(u32x4*)&Ks[buf_][key * KST + dc * 8] = rk[i];                                \
      }                                                                                \
    }                                                                                  \
    _Pragma("unroll") for (int i = 0; i < V_IT; ++i) {                                 \
      const int c = tid + 256 * i;                                                     \
      if (c < DH * 8) *(u32x4*)&Vs[buf_][(c >> 3) * VST + (c & 7) * 8] = rv[i];        \
    }                                                                                  \
  } while (0)

  float m_run = -INFINITY, l_run = 0.f;
  f32x16 oacc[DT];
#pragma unroll
  for (int t = 0; t < DT; ++t) oacc[t] = f32x16{};

  // One key tile: S^T = K Q^T, online softmax, O^T += V^T P^T.
  auto tile = [&](const int buf, const int kv0) {
    f32x16 sacc[2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      sacc[kt] = f32x16{};
#pragma unroll
      for (int s = 0; s < DHP / 16; ++s) {
        bf16x8 kf = *(const bf16x8*)&Ks[buf][(kt * 32 + r32) * KST + s * 16 + g * 8];
        sacc[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[s], sacc[kt], 0, 0, 0);
      }
    }
    // scale into the log2 domain, mask keys past the end, online softmax.
    float mloc = -INFINITY;
    const bool tail = kv0 + BKV > Tj;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        float sv = sacc[kt][e] * a.scale_log2;
        if (tail) {
          const int key = kv0 + kt * 32 + (e >> 2) * 8 + g * 4 + (e & 3);
          if (key >= Tj) sv = -INFINITY;
        }
        sacc[kt][e] = sv;
        mloc = fmaxf(mloc, sv);
      }
    mloc = fmaxf(mloc, other_half(mloc));
    const float m_new = fmaxf(m_run, mloc);
    const float alpha = exp2f(m_run - m_new);
    float lsum = 0.f;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float p = exp2f(sacc[kt][e] - m_new);
        sacc[kt][e] = p;
        lsum += p;
      }
    l_run = l_run * alpha + lsum;
    m_run = m_new;
#pragma unroll
    for (int t = 0; t < DT; ++t) oacc[t] *= alpha;

    // O^T += V^T P^T over four 16-key chunks.
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int kt = c >> 1, jb = (c & 1) * 2;
      u32x4 pw;
      pw[0] = pack_bf16x2(sacc[kt][jb * 4 + 0], sacc[kt][jb * 4 + 1]);
      pw[1] = pack_bf16x2(sacc[kt][jb * 4 + 2], sacc[kt][jb * 4 + 3]);
      pw[2] = pack_bf16x2(sacc[kt][jb * 4 + 4], sacc[kt][jb * 4 + 5]);
      pw[3] = pack_bf16x2(sacc[kt][jb * 4 + 6], sacc[kt][jb * 4 + 7]);
      const bf16x8 pb = __builtin_bit_cast(bf16x8, pw);
#pragma unroll
      for (int t = 0; t < DT; ++t) {
        const bf16_t* vrow = &Vs[buf][(t * 32 + r32) * VST + c * 16 + g * 4];
        const u32x2 lo = *(const u32x2*)vrow;
        const u32x2 hi = *(const u32x2*)(vrow + 8);
        const u32x4 vw = {lo[0], lo[1], hi[0], hi[1]};
        oacc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, vw), pb, oacc[t], 0, 0, 0);
      }
    }
  };

  // The last tile is peeled so the in-loop prefetch is unconditional.
  const int nkv = (Tj + BKV - 1) / BKV;
  ATT_GLOAD(0);
  ATT_LSTORE(0);
  __syncthreads();
  for (int it = 0; it + 1 < nkv; ++it) {
    const int buf = it & 1;
    ATT_GLOAD((it + 1) * BKV);
    __builtin_amdgcn_sched_barrier(0);
    tile(buf, it * BKV);
    __builtin_amdgcn_sched_barrier(0);
    ATT_LSTORE(buf ^ 1);
    __syncthreads();
  }
  tile((nkv - 1) & 1, (nkv - 1) * BKV);
#undef ATT_GLOAD
#undef ATT_LSTORE

  const float l_tot = l_run + other_half(l_run);
  const float inv = 1.0f / l_tot;
  if (qrow < Tj) {
    const long orow = qrow < a.T_img ? (long)b * a.T_img + qrow
                                     : (long)a.B * a.T_img + (long)b * a.T_txt + (qrow - a.T_img);
    bf16_t* op = (bf16_t*)a.o + orow * a.D + h * DH;
#pragma unroll
    for (int t = 0; t < DT; ++t)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const int d = t * 32 + jj * 8 + g * 4;
        if (d < DH) {
          u32x2 w;
          w[0] = pack_bf16x2(oacc[t][jj * 4 + 0] * inv, oacc[t][jj * 4 + 1] * inv);
          w[1] = pack_bf16x2(oacc[t][jj * 4 + 2] * inv, oacc[t][jj * 4 + 3] * inv);
          *(u32x2*)(op + d) = w;
        }
      }
  }
}

hipError_t launch_attn_bf16(const AttnArgs& a, int head_dim, hipStream_t st) {
  dim3 grid((a.Tj + 127) / 128, a.H, a.B), block(256);
  switch (head_dim) {
    case 64: hipLaunchKernelGGL((attn_bf16_kernel<64>), grid, block, 0, st, a); break;
    case 72: hipLaunchKernelGGL((attn_bf16_kernel<72>), grid, block, 0, st, a); break;
    case 128: hipLaunchKernelGGL((attn_bf16_kernel<128>), grid, block, 0, st, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace ditmi
