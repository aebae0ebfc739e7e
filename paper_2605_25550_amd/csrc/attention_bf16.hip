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
// transposed (v^T [dh][T], written that way by the QKV GEMM epilogue, with the
// keys of every 16-key group stored in the order of that permutation,
// kernels.h v_key_pos), so its A operand is one 16-byte LDS read per lane.
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
// head_dim 72 uses q and k rows padded to 80 (written that way by the QKV
// epilogue: zeros, except k's column 72 = 1) for the k-steps of 16, and 96
// rows of V^T (rows 72..95 kept in LDS only).  The pipelined kernel below uses
// that padding to move softmax bookkeeping into the MFMAs (AttnCfg::FOLD).
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
  // Softmax bookkeeping folded into the MFMAs (head_dim 72: padding column
  // DH of k holds 1, so q's column DH carries -m_run into S^T; padding row DH
  // of V^T holds ones, so O^T row DH accumulates the row sum l).
  static constexpr bool FOLD = DHP > DH && VROWS > DH + 4 && DH % 32 % 8 < 4;
  static constexpr int QS = DH / 16, QG = (DH % 16) / 8, QE = DH % 8;  // q register slot of column DH
  static constexpr int LT = DH / 32, LG = (DH % 32) % 8 / 4, LE = (DH % 32) / 8 * 4 + DH % 4;  // O^T slot of row DH
  // ring depth of the pipelined kernel (measured: deeper rings, where they
  // fit, were not faster)
  static constexpr int PIPE_ST = 4;
};


template <int DH, int NW, int QT>
__global__ __launch_bounds__(NW * 64, QT == 1 ? 8 / NW : 1) void attn_bf16_dma_kernel(AttnArgs a) {
  using C = AttnCfg<DH>;
  constexpr bool FOLD = C::FOLD;  // softmax bookkeeping in the MFMAs, as in the pipelined kernel below
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
  // and feed discarded O^T rows: zero in every slot, except row DH, all
  // ones with FOLD (O^T row DH = the row sum l).
  if (C::VROWS > DH) {
    for (int e = tid; e < C::STAGES * (C::VROWS - DH) * 32; e += NW * 64) {
      const int sl = e / ((C::VROWS - DH) * 32), w = e % ((C::VROWS - DH) * 32);
      ((uint32_t*)(smem + sl * C::SLOT + C::KTILE + DH * 128))[w] = FOLD && w < 32 ? 0x3F803F80u : 0u;
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
  // keys 16c+4g+0..3 and 16c+8+4g+0..3 form logical chunk 2c+g of a V^T row
  // (v_key_pos order), so each PV operand is one 16-byte read
  int v_off[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) v_off[c] = C::KTILE + r32 * 128 + (((2 * c + g) ^ C::swz_v(r32)) << 4);

  const float sc = a.scale_log2;
  // Lazy max: probabilities are exp2(s*scale - m_run) <= 2^TAU; bf16 and fp32
  // hold 2^64 exactly in range, and O^T / l sums stay far from fp32 overflow.
  // With FOLD the product already subtracts m_run (0 before the first tile).
  const float TAU = 64.0f;
  float m_run[QT], l_run[QT];
  f32x16 oacc[QT][C::DT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    m_run[qt] = FOLD ? 0.f : -INFINITY;
    l_run[qt] = 0.f;
  }
  bool first = true;
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
          const int kp = v_key_pos(key);
          const int off = C::KTILE + d * 128 + (((kp >> 3) ^ C::swz_v(d)) << 4) + (kp & 7) * 2;
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
      if (FOLD) {
        // scores are relative to m_run already; the running max moves as in
        // the pipelined kernel, kept exactly representable in bf16
        mloc = max_halves(mloc);
        if (first || __builtin_amdgcn_ballot_w64(mloc > TAU) != 0) {
          const float m_new = bf2f(f2bf(m_run[qt] + (first ? mloc : fmaxf(mloc, 0.f))));
          const float delta = m_new - m_run[qt];
          // O and l are still zero at the first tile, whose max may lie far
          // below 0 (exp2(-delta) = inf there, and 0 * inf is NaN)
          const float alpha = first ? 1.0f : __builtin_amdgcn_exp2f(-delta);
#pragma unroll
          for (int t = 0; t < C::DT; ++t) oacc[qt][t] *= alpha;
#pragma unroll
          for (int kt = 0; kt < 2; ++kt) sacc[qt][kt] -= delta;
          m_run[qt] = m_new;
          if (g == C::QG) qf[qt][C::QS][C::QE] = __builtin_bit_cast(__bf16, f2bf(-m_new));
        }
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int e = 0; e < 16; ++e) sacc[qt][kt][e] = __builtin_amdgcn_exp2f(sacc[qt][kt][e]);
      } else {
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
      }
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
          const u32x4 vw = *(const u32x4*)(slot + t * 32 * 128 + v_off[c]);
          oacc[qt][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, vw),
                                                                 __builtin_bit_cast(bf16x8, pw[qt][c]), oacc[qt][t], 0, 0, 0);
        }
    }
    first = false;
  }
  wait_vmcnt<0>();

#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const int qrow = q0 + qt * 32 + r32;
    const float l_tot = sum_halves(FOLD ? (g == C::LG ? oacc[qt][C::LT][C::LE] : 0.f) : l_run[qt]);
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

// Software-pipelined variant (one 32-query tile per wave).  Within a wave,
// the QK^T MFMAs of key tile j+1 are issued between the softmax instructions
// of tile j, and the PV MFMAs of tile j between the row-max instructions of
// tile j+1, so the matrix pipe and the VALU work at the same time even while
// the workgroup barrier keeps the two waves of a SIMD in step.  K of tile
// j+1 is read one iteration earlier than V of tile j, so the ring has four
// slots (tile t of the unit's range [t0, t1) in slot (t - t0) % 4, refilled
// with t + 4 after the barrier that ends iteration t), which keeps two
// iterations between a tile's DMA and its first read.  The loop is unrolled
// four times, so that in each copy the slots are constants.
// The kernel is bound by its VALU work rather than by the matrix pipe
// (measured: removing the 16 row-sum dot products of a tile shortened the
// video DiT attention by 6.5%, the 16 row-max instructions by 3%), so work
// is moved off the VALU where the matrix pipe or the instruction encoding
// can take it: the row sums go through small MFMAs, and LDS addresses are
// lane offsets plus immediates.
template <int DH, int NW, int ST = AttnCfg<DH>::PIPE_ST, int WPC = 1>
__global__ __launch_bounds__(NW * 64, WPC) void attn_bf16_pipe_kernel(AttnArgs a) {
  using C = AttnCfg<DH>;
  constexpr bool FOLD = C::FOLD;
  static_assert(ST == 4 && WPC * (ST * C::SLOT + 1024) <= 160 * 1024, "ring fits the LDS");
  // LDS: the K tiles of the four slots, then their V^T tiles (so that the
  // largest slot offset of each fits a DS instruction's 16-bit immediate),
  // then the spare line.  With constant slots every fragment read is a lane
  // offset plus an immediate, no address arithmetic per tile (measured:
  // video DiT attention -3.7%, joint -1.5%).
  static_assert(ST * C::KTILE <= 65536 && ST * C::VTILE <= 65536, "slot offsets fit the 16-bit LDS immediate");
  constexpr int IPW = (C::TDMA + NW - 1) / NW;  // DMA instructions per wave per tile (uniform)
  __shared__ __attribute__((aligned(1024))) unsigned char smem[ST * C::SLOT + 1024];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 5, r32 = lane & 31;
  // Work item (query block, head, sample), query block fastest, taken in
  // contiguous ranges per XCD: the workgroups an XCD runs at once are query
  // blocks of the same head and share its K and V tiles in that XCD's L2.
  // Units of a split item (the last, partial round) come after the whole
  // items; consecutive units are the same key range of consecutive items.
  const int Tj = a.Tj, Tjp = a.Tj_pad;
  const int nqb = (Tj + NW * 32 - 1) / (NW * 32);
  const int nkv = (Tj + C::BKV - 1) / C::BKV;
  int item, t0 = 0, t1 = nkv, unit = -1;
  if ((int)blockIdx.x < a.n_full) {
    item = xcd_remap(blockIdx.x, a.n_full);
  } else {
    unit = xcd_remap(blockIdx.x - a.n_full, a.n_tail * a.split);
    const int part = unit / a.n_tail;
    item = a.n_full + (unit - part * a.n_tail);
    t0 = nkv * part / a.split;
    t1 = nkv * (part + 1) / a.split;
  }
  const int qb = item % nqb, bh_i = item / nqb;
  const int h = bh_i % a.H, b = bh_i / a.H;
  const long bh = bh_i;
  const bf16_t* __restrict__ qp = (const bf16_t*)a.q + bh * Tj * C::DHP;
  const bf16_t* __restrict__ kp = (const bf16_t*)a.k + bh * Tj * C::DHP;
  const bf16_t* __restrict__ vp = (const bf16_t*)a.v + bh * DH * (long)Tjp;
  const unsigned lds0 = __builtin_amdgcn_readfirstlane(lds_address(smem));
  const int q0 = qb * (NW * 32) + wave * 32;  // first query of this wave

  // DMA of one tile (K and V^T as in the kernel above) into a slot.  The
  // sources are a scalar base (the tile's first K row / V^T column) plus a
  // 32-bit lane offset, fixed for every full tile; only a tile reaching past
  // Tj clamps (K rows past the end re-read row Tj-1, V^T chunks past Tj_pad
  // re-read the last chunk).  Spare instructions re-read instruction 0's K
  // rows into a scratch line, keeping the per-wave DMA count uniform.
  auto dma_off = [&](int t, int rmax, int cmax) -> unsigned {
    const int qi = (t < 0 ? 0 : t) * NW + wave, byte = qi * 1024 + lane * 16;
    if (qi < C::KDMA || t < 0) {
      const int R = byte / C::KROW, pos = (byte % C::KROW) >> 4;
      return (unsigned)(min(R, rmax) * (C::DHP * 2) + (pos ^ C::swz_k(R)) * 16);
    }
    const int vb = byte - C::KTILE, d = vb >> 7, pos = (vb & 127) >> 4;
    return (unsigned)((d * Tjp + min((pos ^ C::swz_v(d)) * 8, cmax)) * 2);
  };
  // Lane offsets of a full tile and of the last tile (clamped where it is
  // partial).
  const int kv_last = (nkv - 1) * C::BKV;
  unsigned doff[IPW], doff_last[IPW];
#pragma unroll
  for (int t = 0; t < IPW; ++t) {
    const int tt = wave + NW * t < C::TDMA ? t : -1;
    doff[t] = dma_off(tt, C::BKV, C::BKV);
    doff_last[t] = dma_off(tt, Tj - 1 - kv_last, Tjp - 8 - kv_last);
  }
  // DMA instruction t of `tile` into slot `slot`.  Past the last tile it
  // re-reads the last tile into the spare line, so that every wave issues
  // the same number of DMA instructions per iteration whatever the tile
  // count, and the vmcnt waits are constants.
  auto issue_one = [&](int tile, int slot, int t) {
    const int qi = wave + NW * t;  // wave-uniform
    const int tl = min(tile, t1 - 1), kv0 = tl * C::BKV;
    const bf16_t* kb = kp + (long)kv0 * C::DHP;  // wave-uniform
    const bf16_t* vb = vp + kv0;
    const bool kpart = qi < C::KDMA || qi >= C::TDMA;
    const unsigned off = tl == nkv - 1 ? doff_last[t] : doff[t];
    const unsigned dst = tile < t1 && qi < C::TDMA
                             ? lds0 + (unsigned)(qi < C::KDMA ? slot * C::KTILE + qi * 1024
                                                              : ST * C::KTILE + slot * C::VTILE + (qi - C::KDMA) * 1024)
                             : lds0 + (unsigned)(ST * C::SLOT);
    dma_16s(kpart ? (const void*)kb : (const void*)vb, off, dst);
  };
  auto issue = [&](int tile) {
#pragma unroll
    for (int t = 0; t < IPW; ++t) issue_one(tile, (tile - t0) % ST, t);
  };
  // V^T columns of keys past the end (last tile only) hold stale workspace
  // bytes; zero them so that their zero probabilities cannot meet a NaN.
  auto zero_v_tail = [&](int tile) {
    const int kv0 = tile * C::BKV, nvalid = Tj - kv0;
    unsigned char* sl = smem + ST * C::KTILE + ((tile - t0) % ST) * C::VTILE;
    for (int e = tid; e < DH * C::BKV; e += NW * 64) {
      const int d = e / C::BKV, key = e % C::BKV;
      const int kp = v_key_pos(key);
      if (key >= nvalid) *(bf16_t*)(sl + d * 128 + (((kp >> 3) ^ C::swz_v(d)) << 4) + (kp & 7) * 2) = 0;
    }
  };

  // V^T rows past head_dim (head_dim 72 only) are never written by the DMA.
  // They are zero, except row DH, which is all ones where the row sums are
  // folded into the PV product (O^T row DH = sum of the tile's P).
  if (C::VROWS > DH) {
    for (int e = tid; e < ST * (C::VROWS - DH) * 32; e += NW * 64) {
      const int sl = e / ((C::VROWS - DH) * 32), w = e % ((C::VROWS - DH) * 32);
      ((uint32_t*)(smem + ST * C::KTILE + sl * C::VTILE + DH * 128))[w] = FOLD && w < 32 ? 0x3F803F80u : 0u;
    }
  }

  bf16x8 qf[C::KS];
  {
    const int qrow = q0 + r32;
#pragma unroll
    for (int s = 0; s < C::KS; ++s)
      qf[s] = qrow < Tj ? *(const bf16x8*)(qp + (long)qrow * C::DHP + s * 16 + g * 8) : bf16x8{};
  }
  int k_off[C::KS];
#pragma unroll
  for (int s = 0; s < C::KS; ++s) k_off[s] = r32 * C::KROW + (((2 * s + g) ^ C::swz_k(r32)) << 4);
  int v_off[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) v_off[c] = ST * C::KTILE + r32 * 128 + (((2 * c + g) ^ C::swz_v(r32)) << 4);

  // k arrives in the exp2 domain (stored pre-scaled by the QKV epilogue).
  // The running max m_run is subtracted inside the QK^T product, so the MFMA
  // result is directly the exp2 argument: with FOLD, k's padding column DH
  // holds 1 and q's holds -m_run (kept exactly representable in bf16);
  // otherwise every S^T accumulator starts at -m_run.
  const float TAU = 64.0f;  // lazy max, as in the kernel above
  float m_run = 0.f;
  // Row sums l of the bf16 probabilities (the same values the PV product
  // multiplies), accumulated on the matrix pipe: a 4x4x4 MFMA with an A
  // operand of ones adds the four bf16 values of each lane's B operand into
  // every element of that lane's accumulator (the VALU is the busier unit).
  // With FOLD the PV product itself carries l.
  f32x4 lacc = f32x4{};
  typedef short i16x4 __attribute__((ext_vector_type(4)));
  const i16x4 ones4 = {0x3F80, 0x3F80, 0x3F80, 0x3F80};
  bool first = true;
  f32x16 oacc[C::DT];
#pragma unroll
  for (int t = 0; t < C::DT; ++t) oacc[t] = f32x16{};
  // Accumulator operand of each tile's first QK^T MFMAs: -m_run in every
  // element (zero with FOLD, where the product subtracts m_run itself).  The
  // MFMA reads it as its C operand and writes S^T elsewhere, so the block is
  // set only when m_run moves, not copied into the accumulators every tile.
  f32x16 sinit = f32x16{};

  // s_mask sets the scores of keys past the end to -inf.
  auto s_mask = [&](int kv0, f32x16 (&s)[2]) {
    if (kv0 + C::BKV > Tj) {
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int e = 0; e < 16; ++e)
          if (kv0 + kt * 32 + (e >> 2) * 8 + g * 4 + (e & 3) >= Tj) s[kt][e] = -INFINITY;
    }
  };
  auto qk = [&](int tile, f32x16 (&s)[2]) {
    const unsigned char* sl = smem + ((tile - t0) % ST) * C::KTILE;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int st = 0; st < C::KS; ++st) {
        const bf16x8 kf = *(const bf16x8*)(sl + kt * 32 * C::KROW + k_off[st]);
        s[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[st], st == 0 ? sinit : s[kt], 0, 0, 0);
      }
  };
  auto rowmax = [&](const f32x16 (&s)[2]) {
    float m = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int e = 0; e < 16; ++e) m = fmaxf(m, s[kt][e]);
    return max_halves(m);
  };

  // prologue: tiles 0 .. ST-2 in flight (tile ST-1 is issued in the first
  // iteration); tiles 0 and 1 landed before the loop
#pragma unroll
  for (int t = 0; t < ST - 1; ++t) issue(t0 + t);
  wait_vmcnt<(ST - 3) * IPW>();
  __syncthreads();
  // the sequence's last tile, where this unit's range holds it, has landed
  // already (else: zeroed at the end of iteration nkv-3)
  if (t1 == nkv && nkv - 1 <= t0 + 1) {
    zero_v_tail(nkv - 1);
    __syncthreads();
  }
  f32x16 sa[2], sb[2];
  qk(t0, sa);
  float mcur = rowmax(sa);

  // One key tile: the exponentials of scur (tile j) and the QK^T of tile
  // j+1 into snext.  The loop runs it twice per trip with the roles of the
  // two score blocks exchanged, so no score block is ever copied.
  auto tile_step = [&](const int j, const int sj, f32x16 (&scur)[2], f32x16 (&snext)[2]) __attribute__((always_inline)) {
    // Keys past the end (last tile only) are masked just before their
    // exponentials.  Their K rows repeat row Tj-1, so the unmasked row max
    // taken earlier is still the max over real keys.
    s_mask(j * C::BKV, scur);
    // lazy rescale for tile j (mcur is its row max relative to m_run): the
    // first tile sets the max; later, only a lead of more than TAU moves it
    // (then O^T, l and the tile's scores shift by the lead)
    if (first || __builtin_amdgcn_ballot_w64(mcur > TAU) != 0) {
      float m_new = m_run + (first ? mcur : fmaxf(mcur, 0.f));
      if (FOLD) m_new = bf2f(f2bf(m_new));  // enters the product as a bf16 operand
      const float delta = m_new - m_run;     // exact
      // O and l are still zero at the first tile, whose max may lie far below
      // 0 (exp2(-delta) = inf there, and 0 * inf is NaN)
      const float alpha = first ? 1.0f : __builtin_amdgcn_exp2f(-delta);
      if (!FOLD) lacc *= alpha;
#pragma unroll
      for (int t = 0; t < C::DT; ++t) oacc[t] *= alpha;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) scur[kt] -= delta;
      m_run = m_new;
      if (FOLD && g == C::QG) qf[C::QS][C::QE] = __builtin_bit_cast(__bf16, f2bf(-m_run));
      if (!FOLD)
#pragma unroll
        for (int e = 0; e < 16; ++e) sinit[e] = -m_run;
      first = false;
    }
    // Softmax of tile j interleaved by hand with the QK^T MFMAs of tile j+1
    // (unconditional: the last iteration reads the next slot's stale K and
    // computes unused scores):
    // K fragments are read two MFMAs ahead, the MFMAs alternate between the
    // two 32-key halves (independent accumulators), and each MFMA is
    // followed by its share of the exponentials.
    u32x4 pw[4];
    // V^T fragments of tile j (landed long before): the first two are read
    // during the last QK^T MFMAs, so the PV product starts without waiting.
    const unsigned char* slv = smem + sj * C::VTILE;  // V^T of tile j (v_off holds the region base)
    constexpr int NP = 4 * C::DT;  // PV MFMAs per tile; MFMA i: key chunk i / DT, O^T tile i % DT
    // The exponentials are split between the two phases: those of the first
    // EX / 8 key chunks (the lane's first EX scores) run beside the QK^T
    // MFMAs, the rest beside the first NPRE PV MFMAs, which read only those
    // first chunks.  Both waves of a SIMD are in the same phase at the same
    // time, so this evens out the VALU work between the phases (measured with
    // 16 of 32 against all 32 after the QK^T product: video DiT attention
    // -2.7%, joint -2%, DiT-XL/2 at 1024 tokens -1.5%; with the row sums on
    // the matrix pipe, 24 of 32 beside the QK^T MFMAs: video DiT -1.5%, joint
    // -1.1%; head_dim 72, whose PV phase carries no row sums, keeps 16).
    constexpr int EX = FOLD ? 16 : 24;
    constexpr int NPRE = EX / 8 * C::DT;  // PV MFMAs before the first one on chunk EX / 8
    constexpr int ND = 3;  // PV MFMAs issued after the barrier
    auto vread = [&](int i) {
      const int c = i / C::DT, t = i % C::DT;
      return *(const u32x4*)(slv + t * 32 * 128 + v_off[c]);
    };
    u32x4 vf[3];
    {
      // K of tile j+1 (in the last iteration a stale slot, read but unused)
      const unsigned char* sln = smem + ((sj + 1) % ST) * C::KTILE;
      constexpr int NQ = 2 * C::KS;  // QK^T MFMAs per tile; MFMA i: half i % 2, k-step i / 2
      auto kread = [&](int i) { return *(const bf16x8*)(sln + (i & 1) * 32 * C::KROW + k_off[i >> 1]); };
      bf16x8 kf[3];
      kf[0] = kread(0);
      kf[1] = kread(1);
#pragma unroll
      for (int i = 0; i < NQ; ++i) {
        if (i + 2 < NQ) kf[(i + 2) % 3] = kread(i + 2);
        snext[i & 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[i % 3], qf[i >> 1], i < 2 ? sinit : snext[i & 1],
                                                               0, 0, 0);
        if (i == NQ - 2) vf[0] = vread(0);
        if (i == NQ - 1) vf[1] = vread(1);

#pragma unroll
        for (int e = i * EX / NQ; e < (i + 1) * EX / NQ; ++e)
          scur[e >> 4][e & 15] = __builtin_amdgcn_exp2f(scur[e >> 4][e & 15]);
        // each pair of probabilities is packed to bf16 as soon as both exist:
        // scores 2p and 2p+1 of the lane's 32 (half p / 8) form word p % 4 of
        // the B operand of the PV MFMAs over key chunk p / 4
#pragma unroll
        for (int p = 0; p < EX / 2; ++p)
          if (2 * p + 1 >= i * EX / NQ && 2 * p + 1 < (i + 1) * EX / NQ)
            pw[p >> 2][p & 3] = pack_bf16x2(scur[p >> 3][(2 * p) & 15], scur[p >> 3][(2 * p + 1) & 15]);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    // PV of tile j (consecutive MFMAs on different O^T tiles), V^T read two
    // MFMAs ahead, interleaved with the row max of tile j+1.  The DMA of tile
    // j+ST-1 into the slot of tile j-1 (released by the last barrier) is
    // spread over the same sequence, one instruction every few MFMAs: issued
    // as a burst after the barrier, the workgroup's DMA instructions queue at
    // the address unit and stall the waves at issue.  Placed here rather than
    // beside the QK^T MFMAs, which carry most of the exponentials, it measured
    // video DiT attention -1%, DiT-XL/2 at 1024 tokens -1.6%.
    {
      float m = -INFINITY;
#pragma unroll
      for (int i = 0; i < NP; ++i) {
        if (i + 2 < NP) vf[(i + 2) % 3] = vread(i + 2);
#pragma unroll
        for (int t = 0; t < IPW; ++t)
          if (i == t * (NP - ND) / IPW) issue_one(j + ST - 1, (sj + ST - 1) % ST, t);
        if (i < NP - ND)
          oacc[i % C::DT] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, vf[i % 3]),
                                                                    __builtin_bit_cast(bf16x8, pw[i / C::DT]),
                                                                    oacc[i % C::DT], 0, 0, 0);
#pragma unroll
        for (int e = i * 32 / NP; e < (i + 1) * 32 / NP; ++e) m = fmaxf(m, snext[e >> 4][e & 15]);
        // exponentials and packing of chunks EX / 8 .. 3
        if (i < NPRE) {
#pragma unroll
          for (int e = EX + i * (32 - EX) / NPRE; e < EX + (i + 1) * (32 - EX) / NPRE; ++e)
            scur[e >> 4][e & 15] = __builtin_amdgcn_exp2f(scur[e >> 4][e & 15]);
#pragma unroll
          for (int p = EX / 2; p < 16; ++p)
            if (2 * p + 1 >= EX + i * (32 - EX) / NPRE && 2 * p + 1 < EX + (i + 1) * (32 - EX) / NPRE)
              pw[p >> 2][p & 3] = pack_bf16x2(scur[p >> 3][(2 * p) & 15], scur[p >> 3][(2 * p + 1) & 15]);
        }
        // row sum of the tile's 32 probabilities of this lane: eight 4x4x4
        // MFMAs of two packed words each, spread over the PV MFMAs
        if (!FOLD)
#pragma unroll
          for (int k = 0; k < 8; ++k)
            if (i == (k * NP + NP - 1) / 8) {
              const u32x2 two = {pw[k >> 1][(k & 1) * 2], pw[k >> 1][(k & 1) * 2 + 1]};
              lacc = __builtin_amdgcn_mfma_f32_4x4x4bf16_1k(ones4, __builtin_bit_cast(i16x4, two), lacc, 0, 0, 0);
            }
        __builtin_amdgcn_sched_barrier(0);
      }
      mcur = max_halves(m);
    }
    // tile j+2 must have landed for every wave before the next iteration's
    // QK^T (tiles j+3 .. j+ST-1 may still be in flight), and every wave must
    // be done with the slot of tile j before it takes tile j+ST
    wait_vmcnt<(ST - 3) * IPW>();
    __syncthreads();
    // the last ND PV MFMAs of the tile, on fragments already in registers
    // (the barrier's fence has waited for their LDS reads): the matrix pipe
    // has work while the next tile's first K fragments load (measured: video
    // DiT attention -2.5%, joint -1.5%, DiT-XL/2 at 1024 tokens -2%; deferring
    // four or six instead is no faster)
#pragma unroll
    for (int i = NP - ND; i < NP; ++i)
      oacc[i % C::DT] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, vf[i % 3]),
                                                                __builtin_bit_cast(bf16x8, pw[i / C::DT]),
                                                                oacc[i % C::DT], 0, 0, 0);
    if (t1 == nkv && j + 2 == nkv - 1) {  // the last tile's V^T is read in iteration nkv-1
      zero_v_tail(nkv - 1);
      __syncthreads();
    }
  };
  int j = t0;
  for (; j + 3 < t1; j += 4) {
    tile_step(j, 0, sa, sb);
    tile_step(j + 1, 1, sb, sa);
    tile_step(j + 2, 2, sa, sb);
    tile_step(j + 3, 3, sb, sa);
  }
  if (j < t1) tile_step(j, 0, sa, sb);
  if (j + 1 < t1) tile_step(j + 1, 1, sb, sa);
  if (j + 2 < t1) tile_step(j + 2, 2, sa, sb);
  wait_vmcnt<0>();

  {
    const int qrow = q0 + r32;
    // with FOLD, l is O^T row DH: element LE of tile LT in the lanes of half
    // LG (the other half holds a zero row there)
    const float l_lane = FOLD ? (g == C::LG ? oacc[C::LT][C::LE] : 0.f) : lacc[0];
    const float l_tot = sum_halves(l_lane);
    if (unit >= 0) {
      // a unit of a split item: O relative to its own m_run, m_run and l,
      // for attn_merge
      if (qrow < Tj) {
        float* pr = a.part + ((long)unit * (NW * 32) + wave * 32 + r32) * (DH + 4);
#pragma unroll
        for (int t = 0; t < C::DT; ++t)
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) {
            const int d = t * 32 + jj * 8 + g * 4;
            if (d < DH)
              *(f32x4*)(pr + d) = f32x4{oacc[t][jj * 4 + 0], oacc[t][jj * 4 + 1], oacc[t][jj * 4 + 2],
                                        oacc[t][jj * 4 + 3]};
          }
        if (g == 0) *(f32x2*)(pr + DH) = f32x2{m_run, l_tot};
      }
      return;
    }
    const float inv = 1.0f / l_tot;
    if (qrow < Tj) {
      const long orow = qrow < a.T_img ? (long)b * a.T_img + qrow
                                       : (long)a.B * a.T_img + (long)b * a.T_txt + (qrow - a.T_img);
      bf16_t* op = (bf16_t*)a.o + orow * a.D + h * DH;
      // Lane half g holds columns 8 jj + 4 g .. +3 of each O^T tile.  For a
      // pair of 8-column groups (jj, jj+1) a swap between the halves gives
      // half 0 columns 0..7 of the pair and half 1 columns 8..15, so each
      // lane stores 16 contiguous bytes and a row's 32 bytes come from one
      // instruction.
#pragma unroll
      for (int t = 0; t < C::DT; ++t)
#pragma unroll
        for (int jp = 0; jp < 2; ++jp) {
          const int d0 = t * 32 + jp * 16;
          auto word = [&](int jj, int k) {
            return pack_bf16x2(oacc[t][jj * 4 + 2 * k] * inv, oacc[t][jj * 4 + 2 * k + 1] * inv);
          };
          if (d0 + 16 <= DH) {
            u32x4 w;
#pragma unroll
            for (int k = 0; k < 2; ++k) {
              const auto r = __builtin_amdgcn_permlane32_swap(word(2 * jp, k), word(2 * jp + 1, k), false, false);
              w[k] = r[0];
              w[2 + k] = r[1];
            }
            *(u32x4*)(op + d0 + g * 8) = w;
          } else {
#pragma unroll
            for (int jj = 2 * jp; jj < 2 * jp + 2; ++jj) {
              const int d = t * 32 + jj * 8 + g * 4;
              if (d < DH) *(u32x2*)(op + d) = u32x2{word(jj, 0), word(jj, 1)};
            }
          }
        }
    }
  }
}

// Merge of the units of the split items: per query, with m = max_s m_s and
// f_s = 2^(m_s - m),  O = sum_s f_s O_s / sum_s f_s l_s  (ranges in order
// s = 0, 1, ...), stored as the o row of the query in bf16.  One lane per
// four columns of one query row.
template <int DH, int QB>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnArgs a) {
  constexpr int G = DH / 4;  // column groups per row
  const long e = blockIdx.x * 256L + threadIdx.x;
  if (e >= (long)a.n_tail * QB * G) return;
  const int c4 = (int)(e % G) * 4;
  const int qr = (int)((e / G) % QB), ti = (int)(e / ((long)G * QB));
  const int item = a.n_full + ti;
  const int nqb = (a.Tj + QB - 1) / QB;
  const int qb = item % nqb, bh = item / nqb, h = bh % a.H, b = bh / a.H;
  const int qrow = qb * QB + qr;
  if (qrow >= a.Tj) return;
  const long stride = (long)a.n_tail * QB * (DH + 4);
  const float* p0 = a.part + ((long)ti * QB + qr) * (DH + 4);
  float m = -INFINITY;
  for (int s = 0; s < a.split; ++s) m = fmaxf(m, p0[s * stride + DH]);
  float den = 0.f;
  f32x4 num = {0.f, 0.f, 0.f, 0.f};
  for (int s = 0; s < a.split; ++s) {
    const float* ps = p0 + s * stride;
    const float f = __builtin_amdgcn_exp2f(ps[DH] - m);
    den += f * ps[DH + 1];
    const f32x4 o = *(const f32x4*)(ps + c4);
    num[0] += f * o[0];
    num[1] += f * o[1];
    num[2] += f * o[2];
    num[3] += f * o[3];
  }
  const float inv = 1.0f / den;
  const long orow = qrow < a.T_img ? (long)b * a.T_img + qrow
                                   : (long)a.B * a.T_img + (long)b * a.T_txt + (qrow - a.T_img);
  bf16_t* op = (bf16_t*)a.o + orow * a.D + h * DH + c4;
  *(u32x2*)op = u32x2{pack_bf16x2(num[0] * inv, num[1] * inv), pack_bf16x2(num[2] * inv, num[3] * inv)};
}

// Items of the pipelined kernel (256 queries each) that fill whole rounds of
// 256 run whole; the items of the last, partial round are split into S key
// ranges when that shortens the launch: the last round then takes
// ceil(n_tail S / 256) / S of a round instead of one, plus ~1% of a round
// per range for the partial stores and the merge.  Each range keeps at
// least 4 key tiles.  Video DiT, 17550 tokens: 1656 items = 6 rounds + 120,
// S = 2; joint DiT, 4352 tokens: 408 = 1 round + 152, S = 5.
static constexpr int ATTN_PIPE_QUERIES = 256;

size_t attn_split_plan(int B, int H, int Tj, int head_dim, size_t part_cap, int* n_full, int* n_tail, int* split) {
  const long items = (long)((Tj + ATTN_PIPE_QUERIES - 1) / ATTN_PIPE_QUERIES) * H * B;
  const int nkv = (Tj + 63) / 64;
  *n_full = (int)items;
  *n_tail = 0;
  *split = 1;
  const long tail = items % 256;
  if (items < 256 || tail == 0) return 0;
  double best = 1.0;
  int best_s = 1;
  for (int S = 2; S <= 8 && nkv / S >= 4; ++S) {
    const size_t bytes = (size_t)S * tail * ATTN_PIPE_QUERIES * (head_dim + 4) * sizeof(float);
    if (bytes > part_cap) break;
    const double cost = (double)((tail * S + 255) / 256) / S + 0.01 * S;
    if (cost < best - 0.05) best = cost, best_s = S;
  }
  if (best_s == 1) return 0;
  *n_full = (int)(items - tail);
  *n_tail = (int)tail;
  *split = best_s;
  return (size_t)best_s * tail * ATTN_PIPE_QUERIES * (head_dim + 4) * sizeof(float);
}

hipError_t launch_attn_bf16(const AttnArgs& a, int head_dim, hipStream_t st) {
  // Enough work items for every CU, or at least half of them with long
  // sequences (32 key tiles or more, where the steady state dominates, e.g.
  // 3 heads over 17550 tokens: 207 items): the pipelined kernel, 8 waves x
  // 32 queries per workgroup.  Otherwise (few, short sequences) the first
  // kernel with 4 waves x 32 queries, which spreads the work over twice as
  // many workgroups.
  const long items = (long)((a.Tj + 255) / 256) * a.H * a.B;
  const bool wide = items >= 256 || (items >= 128 && a.Tj >= 2048);
  const int nw = wide ? 8 : 4;
  dim3 grid((a.Tj + nw * 32 - 1) / (nw * 32), a.H, a.B), block(nw * 64);
  // the pipelined kernel maps a 1-D grid to its items and split units
  AttnArgs p = a;
  if (!wide || !a.part || a.split < 2) {
    p.n_full = (int)(grid.x * grid.y * grid.z);
    p.n_tail = 0;
    p.split = 1;
  }
  dim3 grid1(p.n_full + p.n_tail * p.split);
  const long merge_lanes = (long)p.n_tail * ATTN_PIPE_QUERIES * (head_dim / 4);
  dim3 grid_m((unsigned)((merge_lanes + 255) / 256));
#define ATTN_LAUNCH(DHV)                                                                          \
  if (wide) {                                                                                     \
    hipLaunchKernelGGL((attn_bf16_pipe_kernel<DHV, 8>), grid1, block, 0, st, p);                   \
    if (p.n_tail > 0)                                                                             \
      hipLaunchKernelGGL((attn_merge_kernel<DHV, ATTN_PIPE_QUERIES>), grid_m, dim3(256), 0, st, p); \
  } else {                                                                                        \
    hipLaunchKernelGGL((attn_bf16_dma_kernel<DHV, 4, 1>), grid, block, 0, st, a);                  \
  }
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
