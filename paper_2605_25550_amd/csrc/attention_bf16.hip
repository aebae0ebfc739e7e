// Fused multi-head attention, bf16 operands, fp32 softmax and accumulation,
// for gfx950: O = softmax(q k^T / sqrt(dh)) v per (sample, head), the
// O(T^2 D) part of the DiT block.  Flash-style single pass with an online
// softmax, so no T x T score matrix ever reaches HBM.
//
// Orientation.  Each wavefront owns 32 queries.  It computes S^T = K Q^T with
// v_mfma_f32_32x32x16_bf16 (A = a K fragment from LDS, B = the wave's Q^T held
// in registers for the whole pass), so every lane holds the scores of ONE
// query (its lane index mod 32) for 32 keys: the row max is in-lane plus one
// exchange with the other half-wavefront, and the row sum needs no exchange
// until the end.  The probabilities are then already laid out as the B
// operand of O^T = V^T P^T (keys permuted consistently on both operands), and
// O^T's accumulators again belong to the lane's own query.  V is consumed
// transposed (v^T [dh][T], written that way by the QKV GEMM epilogue), so its
// A operand is two 8-byte LDS reads per lane.
//
// Schedule.  A workgroup is 8 waves (256 queries; 4 waves for small grids),
// two waves per SIMD, so one wave's softmax VALU work runs while the other's
// MFMAs are in the matrix pipe.  K and V^T tiles of 64 keys are copied
// HBM -> LDS by the global_load_lds_dwordx4 DMA path into a ring of 3 slots,
// two tiles ahead of the math; the DMA cannot pad rows, so 16-byte chunks are
// XOR-swizzled per row to keep the fragment reads free of bank conflicts.
// Every wave issues the same number of DMAs per tile (spare ones re-read a
// valid address into a scratch line) so the explicit vmcnt waits are uniform.
//
// Softmax.  Scores are masked by starting the QK^T accumulators at -inf for
// keys past the end (only on the last tile).  exp2 with log2(e)/sqrt(dh)
// folded into one FMA.  The running max is only moved, and O^T and l
// rescaled, when a tile's max exceeds it by more than 2^64 in the exp2
// domain: probabilities stay <= 2^64, exactly representable in bf16 and far
// from overflowing the fp32 sums, so after the first tile the rescale (which
// touches every accumulator) practically never runs.
//
// head_dim 72 uses q and k rows zero-padded to 80 (written that way by the
// QKV epilogue) for the k-steps of 16, and 96 rows of V^T (rows 72..95 zero).
#include "common.h"
#include "kernels.h"

namespace ditmi {

template <int DH>
struct AttnCfg {
  static constexpr int DHP = (DH + 15) / 16 * 16;  // q/k row length in memory (zero padded)
  static constexpr int BKV = 64;
  static constexpr int KROW = DHP * 2;          // bytes per K row in LDS
  static constexpr int KTILE = BKV * KROW;      // bytes
  static constexpr int DT = (DH + 31) / 32;     // 32-row tiles of V^T / O^T
  static constexpr int VROWS = DT * 32;
  static constexpr int VTILE = VROWS * 128;     // V^T: 128 bytes (64 keys) per row
  static constexpr int SLOT = KTILE + VTILE;
  static constexpr int STAGES = 3;
  static constexpr int KS = DHP / 16;           // k-steps of QK^T
  static constexpr int KDMA = KTILE / 1024;     // DMA instructions per tile: K ...
  static constexpr int TDMA = KDMA + DH * 128 / 1024;  // ... plus the real V^T rows
  // XOR masks of the 16-byte chunk index, per row
  static __device__ __forceinline__ int swz_k(int r) {
    return DHP == 128 ? (r & 15) : (DHP == 64 ? ((r >> 1) & 7) : ((r >> 3) & 1));
  }
  static __device__ __forceinline__ int swz_v(int d) { return (d >> 1) & 7; }
  static_assert(KTILE % 1024 == 0 && DH * 128 % 1024 == 0, "tiles are whole 1 KB DMA blocks");
};

template <int DH, int NW, int QT>
__global__ __launch_bounds__(NW * 64, 8 / NW) void attn_bf16_dma_kernel(AttnArgs a) {
  using C = AttnCfg<DH>;
  constexpr int IPW = (C::TDMA + NW - 1) / NW;  // DMA instructions per wave per tile (uniform)
  // ring of slots, then a 1 KB line that absorbs the spare DMAs
  __shared__ __attribute__((aligned(1024))) unsigned char smem[C::STAGES * C::SLOT + 1024];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 5, r32 = lane & 31;
  const int b = blockIdx.z, h = blockIdx.y;
  const int Tj = a.Tj, Tjp = a.Tj_pad;
  const long bh = (long)b * a.H + h;
  const bf16_t* __restrict__ qp = (const bf16_t*)a.q + bh * Tj * C::DHP;
  const bf16_t* __restrict__ kp = (const bf16_t*)a.k + bh * Tj * C::DHP;
  const bf16_t* __restrict__ vp = (const bf16_t*)a.v + bh * DH * (long)Tjp;
  const unsigned lds0 = __builtin_amdgcn_readfirstlane(lds_address(smem));
  const int q0 = blockIdx.x * (NW * QT * 32) + wave * (QT * 32);  // first query of this wave

  // DMA of one tile: instruction qi < KDMA covers K bytes [1024 qi, +1024) of
  // the slot, qi < TDMA the V^T bytes after it; wave w issues qi = w + NW t.
  auto issue = [&](int tile) {
    const int kv0 = tile * C::BKV;
    const unsigned base = lds0 + (unsigned)((tile % C::STAGES) * C::SLOT);
#pragma unroll
    for (int t = 0; t < IPW; ++t) {
      const int qi = wave + NW * t;  // wave-uniform
      const int byte = qi * 1024 + lane * 16;
      const bf16_t* src;
      unsigned dst = base + (unsigned)(qi * 1024);
      if (qi < C::KDMA) {
        const int R = byte / C::KROW, pos = (byte % C::KROW) >> 4;
        const int c = pos ^ C::swz_k(R);
        src = kp + (long)min(kv0 + R, Tj - 1) * C::DHP + c * 8;
      } else if (qi < C::TDMA) {
        const int vb = byte - C::KTILE;
        const int d = vb >> 7, pos = (vb & 127) >> 4;
        const int c = pos ^ C::swz_v(d);
        src = vp + (long)d * Tjp + min(kv0 + c * 8, Tjp - 8);
      } else {  // spare: keeps the per-wave DMA count uniform
        src = kp + lane * 8;
        dst = lds0 + (unsigned)(C::STAGES * C::SLOT);
      }
      dma_16(src, dst);
    }
  };

  // V^T rows past head_dim (head_dim 72 only) are never written by the DMA
  // and feed discarded O^T rows; keep them zero in every slot.
  if (C::VROWS > DH) {
    for (int e = tid; e < C::STAGES * (C::VROWS - DH) * 32; e += NW * 64) {
      const int sl = e / ((C::VROWS - DH) * 32), w = e % ((C::VROWS - DH) * 32);
      ((uint32_t*)(smem + sl * C::SLOT + C::KTILE + DH * 128))[w] = 0u;
    }
  }

  // Q^T fragments for the wave's two query tiles (B operands), zero past the end.
  bf16x8 qf[QT][C::KS];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const int qrow = q0 + qt * 32 + r32;
#pragma unroll
    for (int s = 0; s < C::KS; ++s)
      qf[qt][s] = qrow < Tj ? *(const bf16x8*)(qp + (long)qrow * C::DHP + s * 16 + g * 8) : bf16x8{};
  }

  // LDS read offsets (within a slot) of this lane's K and V^T fragments.  The
  // swizzles depend on the row only through r32, so the second 32-key half of
  // K and the other 32-row tiles of V^T are constant offsets away.
  int k_off[C::KS];
#pragma unroll
  for (int s = 0; s < C::KS; ++s) k_off[s] = r32 * C::KROW + (((2 * s + g) ^ C::swz_k(r32)) << 4);
  int v_lo[4], v_hi[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) {  // keys 16c+4g.. in logical chunk 2c, keys 16c+8+4g.. in chunk 2c+1
    v_lo[c] = C::KTILE + r32 * 128 + (((2 * c) ^ C::swz_v(r32)) << 4) + g * 8;
    v_hi[c] = C::KTILE + r32 * 128 + (((2 * c + 1) ^ C::swz_v(r32)) << 4) + g * 8;
  }

  const float sc = a.scale_log2;
  // Lazy max: probabilities are exp2(s*scale - m_run) <= 2^TAU; bf16 and fp32
  // hold 2^64 exactly in range, and O^T / l sums stay far from fp32 overflow.
  const float TAU = 64.0f;
  float m_run[QT], l_run[QT];
  f32x16 oacc[QT][C::DT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    m_run[qt] = -INFINITY;
    l_run[qt] = 0.f;
  }
#pragma unroll
  for (int qt = 0; qt < QT; ++qt)
#pragma unroll
    for (int t = 0; t < C::DT; ++t) oacc[qt][t] = f32x16{};

  const int nkv = (Tj + C::BKV - 1) / C::BKV;
#pragma unroll
  for (int s = 0; s < C::STAGES - 1; ++s) issue(s);

  for (int it = 0; it < nkv; ++it) {
    const int kv0 = it * C::BKV;
    wait_vmcnt<(C::STAGES - 2) * IPW>();
    __syncthreads();
    issue(it + C::STAGES - 1);  // past the end: clamped re-reads into a free slot
    const unsigned char* slot = smem + (it % C::STAGES) * C::SLOT;
    if (kv0 + C::BKV > Tj) {
      // V^T columns of keys past the end hold stale workspace bytes: zero them.
      const int nvalid = Tj - kv0;
      for (int e = tid; e < DH * C::BKV; e += NW * 64) {
        const int d = e / C::BKV, key = e % C::BKV;
        if (key >= nvalid) {
          const int off = C::KTILE + d * 128 + (((key >> 3) ^ C::swz_v(d)) << 4) + (key & 7) * 2;
          *(bf16_t*)(smem + (it % C::STAGES) * C::SLOT + off) = 0;
        }
      }
      __syncthreads();
    }

    // S^T[key][query] for both query tiles; each K fragment feeds two MFMAs.
    // Accumulators start at 0 for real keys and -inf for keys past the end,
    // so the MFMA itself produces the masked scores.
    // (lane layout: key kv0 + kt*32 + 8*(e/4) + 4*g + e%4)
    f32x16 sacc[QT][2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      f32x16 init = f32x16{};
      if (kv0 + C::BKV > Tj) {
#pragma unroll
        for (int e = 0; e < 16; ++e)
          init[e] = kv0 + kt * 32 + (e >> 2) * 8 + g * 4 + (e & 3) < Tj ? 0.f : -INFINITY;
      }
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) sacc[qt][kt] = init;
    }
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int s = 0; s < C::KS; ++s) {
        const bf16x8 kf = *(const bf16x8*)(slot + kt * 32 * C::KROW + k_off[s]);
#pragma unroll
        for (int qt = 0; qt < QT; ++qt)
          sacc[qt][kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[qt][s], sacc[qt][kt], 0, 0, 0);
      }

    u32x4 pw[QT][4];  // P^T as bf16 B operands, per query tile and 16-key chunk
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      // row max (raw scores; the scale is positive), lazy rescale, exp2, row sum
      float mloc = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          mloc = fmaxf(mloc, sacc[qt][kt][e]);
        }
      mloc = max_halves(mloc) * sc;
      if (m_run[qt] == -INFINITY) {
        m_run[qt] = mloc;  // first tile: O and l are still zero, nothing to rescale
      } else if (__builtin_amdgcn_ballot_w64(mloc > m_run[qt] + TAU) != 0) {
        // rare: a score beyond the running max by more than 2^TAU
        const float m_new = fmaxf(m_run[qt], mloc);
        const float alpha = __builtin_amdgcn_exp2f(m_run[qt] - m_new);
        l_run[qt] *= alpha;
#pragma unroll
        for (int t = 0; t < C::DT; ++t) oacc[qt][t] *= alpha;
        m_run[qt] = m_new;
      }
      const float mneg = -m_run[qt];
      float lsum = 0.f;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const float p = __builtin_amdgcn_exp2f(fmaf(sacc[qt][kt][e], sc, mneg));
          sacc[qt][kt][e] = p;
          lsum += p;
        }
      l_run[qt] += lsum;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int kt = c >> 1, jb = (c & 1) * 2;
        pw[qt][c] = u32x4{pack_bf16x2(sacc[qt][kt][jb * 4 + 0], sacc[qt][kt][jb * 4 + 1]),
                          pack_bf16x2(sacc[qt][kt][jb * 4 + 2], sacc[qt][kt][jb * 4 + 3]),
                          pack_bf16x2(sacc[qt][kt][jb * 4 + 4], sacc[qt][kt][jb * 4 + 5]),
                          pack_bf16x2(sacc[qt][kt][jb * 4 + 6], sacc[qt][kt][jb * 4 + 7])};
      }
      // O^T += V^T P^T; each V^T fragment is read here for this query tile
#pragma unroll
      for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int t = 0; t < C::DT; ++t) {
          const u32x2 lo = *(const u32x2*)(slot + t * 32 * 128 + v_lo[c]);
          const u32x2 hi = *(const u32x2*)(slot + t * 32 * 128 + v_hi[c]);
          const u32x4 vw = {lo[0], lo[1], hi[0], hi[1]};
          oacc[qt][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, vw),
                                                                 __builtin_bit_cast(bf16x8, pw[qt][c]), oacc[qt][t], 0, 0, 0);
        }
    }
  }
  wait_vmcnt<0>();

#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const int qrow = q0 + qt * 32 + r32;
    const float l_tot = sum_halves(l_run[qt]);
    const float inv = 1.0f / l_tot;
    if (qrow < Tj) {
      const long orow = qrow < a.T_img ? (long)b * a.T_img + qrow
                                       : (long)a.B * a.T_img + (long)b * a.T_txt + (qrow - a.T_img);
      bf16_t* op = (bf16_t*)a.o + orow * a.D + h * DH;
#pragma unroll
      for (int t = 0; t < C::DT; ++t)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          const int d = t * 32 + jj * 8 + g * 4;
          if (d < DH)
          *(u32x2*)(op + d) = u32x2{pack_bf16x2(oacc[qt][t][jj * 4 + 0] * inv, oacc[qt][t][jj * 4 + 1] * inv),
                                    pack_bf16x2(oacc[qt][t][jj * 4 + 2] * inv, oacc[qt][t][jj * 4 + 3] * inv)};
        }
    }
  }
}

hipError_t launch_attn_bf16(const AttnArgs& a, int head_dim, hipStream_t st) {
  // 8 waves x 32 queries per workgroup (two waves per SIMD); 4 waves when the
  // grid would otherwise leave CUs idle.
  const bool wide = (long)((a.Tj + 255) / 256) * a.H * a.B >= 256;
  const int nw = wide ? 8 : 4;
  dim3 grid((a.Tj + nw * 32 - 1) / (nw * 32), a.H, a.B), block(nw * 64);
#define ATTN_LAUNCH(DHV)                                                                       \
  if (wide) hipLaunchKernelGGL((attn_bf16_dma_kernel<DHV, 8, 1>), grid, block, 0, st, a);     \
  else hipLaunchKernelGGL((attn_bf16_dma_kernel<DHV, 4, 1>), grid, block, 0, st, a);
  switch (head_dim) {
    case 64: ATTN_LAUNCH(64) break;
    case 72: ATTN_LAUNCH(72) break;
    case 128: ATTN_LAUNCH(128) break;
    default: return hipErrorInvalidValue;
  }
#undef ATTN_LAUNCH
  return hipGetLastError();
}

}  // namespace ditmi
