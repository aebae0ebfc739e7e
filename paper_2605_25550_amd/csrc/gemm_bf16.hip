// bf16 MFMA GEMM for the DiT block's linear layers (QKV, output projection,
// MLP fc1/fc2 and the final layer) on gfx950:
//   y[M, N] = A[M, K] * W[N, K]^T + bias,  fp32 accumulate,
// followed by a fused epilogue (kernels.h: Epi).
//
// Both operands are K-contiguous.  A workgroup of WGM x WGN waves owns a
// BM x BN tile (4 waves for 128- and 64-row tiles, 8 waves, two per SIMD, for
// 256-row tiles); each wave owns (BM/WGM) x (BN/WGN) as 32x32 accumulators
// of v_mfma_f32_32x32x16_bf16, whose lanes each read 8 consecutive bf16 of
// one row from LDS.
//
// Memory pipeline.  K is consumed in 64-wide slices (128 bytes per row, one
// full cache line).  Each slice of A and W is copied HBM -> LDS by the
// global_load_lds_dwordx4 DMA path (no VGPR staging, no ds_write
// instructions) into a ring of STAGES slice buffers.  A DMA instruction moves
// 8 rows x 128 bytes; its address is a scalar base (operand + k offset) plus a
// fixed 32-bit per-lane offset, so the loop spends no vector ALU work on
// addresses.  A slot is refilled as soon as every wave has read its last
// fragments (before the last k-step's MFMAs), so STAGES - 1 slices are in
// flight while one is consumed; the refill's DMA instructions are placed one
// after each MFMA of two k-steps rather than issued as one burst, because the
// address unit takes 16 cycles per 1 KB instruction and a wave waiting to
// issue DMA cannot issue MFMAs.  Rows cannot be padded (the DMA writes 16
// bytes per lane at consecutive LDS addresses); instead the 16-byte chunk c
// of row r is stored at position c ^ f(r), f(r) = (r & 7) ^ ((r >> 3) & 1),
// which keeps the 16 rows read by one quarter-wavefront on distinct banks.
// The compiler does not see the DMA (inline assembly), so the vmcnt waits
// that order it are explicit, and scheduling barriers keep each k-step's
// fragment reads one MFMA group ahead of their use.
//
// Workgroup ids are remapped so that consecutive tiles (sharing A rows) run
// on the same XCD and its L2.  The epilogue stages 32-row slabs of the
// accumulators through LDS so that every global access is a contiguous 8- or
// 16-byte vector per lane.
#include "common.h"
#include "kernels.h"

namespace ditmi {

template <int BM, int BN, int WGM, int WGN, int STAGES>
struct GemmCfg {
  static constexpr int NW = WGM * WGN;          // waves per workgroup (WGM along M, WGN along N)
  static constexpr int BK = 64;                 // K per slice (128 bytes per row)
  static constexpr int WTM = BM / WGM, WTN = BN / WGN;
  static constexpr int TM = WTM / 32, TN = WTN / 32;
  static constexpr int ROWS = BM + BN;          // A rows then W rows in a slice buffer
  static constexpr int SLICE = ROWS * 128;      // bytes per slice buffer
  static constexpr int IPW = ROWS / (8 * NW);   // DMA instructions (8 rows each) per wave per slice
  static constexpr int IPW_A = BM / (8 * NW);   // ... of which read A
  static constexpr int CST = WTN + 4;           // fp32 row stride of an epilogue slab
  static constexpr int LDS_MAIN = STAGES * SLICE;
  static constexpr int LDS_EPI = NW * 32 * CST * 4;
  static constexpr int LDS = LDS_MAIN > LDS_EPI ? LDS_MAIN : LDS_EPI;
  static_assert(WTM % 32 == 0 && WTN % 32 == 0, "wave tiles are multiples of 32");
  static_assert(NW % 2 == 0 && ROWS % (8 * NW) == 0 && BM % (8 * NW) == 0, "uniform DMA split");
  static_assert(STAGES >= 2 && (STAGES - 1) * IPW < 64, "vmcnt range");
  static_assert(LDS <= 160 * 1024, "LDS per CU");
};

// Orders one wave's LDS accesses across its lanes for the compiler (the
// hardware already executes a wave's LDS instructions in order).
__device__ __forceinline__ void wave_lds_fence() { __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront"); }

// Stored position of 16-byte chunk c of slice row r.
__device__ __forceinline__ int chunk_pos(int r, int c) { return c ^ ((r & 7) ^ ((r >> 3) & 1)); }

// Fused epilogue of one wave's strip of WTN columns, applied one 32-row slab
// at a time from fp32 accumulators staged in LDS (row stride CST).  Each lane
// takes four consecutive columns of one row (or, for the v part of the QKV
// projection, one column and four consecutive rows) and uses 8- or 16-byte
// global accesses.  Nothing it reads from global memory is waited for at the
// point of use: the bias (and the gate of the strip's first sample) is
// requested when the kernel starts, and the residual rows of a slab are
// requested before the previous slab is processed, so a slab does not expose
// a memory round trip.
template <int EPI, int WTN, int CST>
struct Epilogue {
  static constexpr int PL = 32 * WTN / 256;  // 4-element groups per lane per slab
  static constexpr int CPR = WTN / 4;        // 4-column groups per slab row
  static constexpr bool RES = EPI == EPI_RESID || EPI == EPI_RESID2;
  static constexpr int NX = RES ? PL : 1;
  // A lane's column group in iteration it is (lane + 64 it) % CPR, which
  // takes NCG distinct values (NCG = 1 when CPR divides 64).
  static constexpr int gcd(int a, int b) { return b == 0 ? a : gcd(b, a % b); }
  static constexpr int NCG = CPR / gcd(64, CPR);
  static_assert(32 * WTN % 256 == 0, "slab must split evenly over 64 lanes");
  static constexpr bool QKV = EPI == EPI_QKV;
  f32x4 bias4[NCG];           // bias of the lane's column groups (row path)
  float vb[QKV ? PL : 1];     // v path: bias of the column of each group
  f32x4 gate4[RES ? NCG : 1]; // EPI_RESID: gate of sample b0 for the lane's column groups
  int b0;
  float inv_rpb;              // 1 / rows_per_batch, for div_exact
  // EPI_QKV, q and k columns: for each column group of the lane, its head's
  // column block of q or k (element h Tj qk_stride + d), the factor it is
  // stored with, and whether it is the head's last group, after which the
  // padding columns are written too (0: no, 1: of q, 2: of k).
  bf16_t* qk_col[QKV ? NCG : 1];
  float qk_f[QKV ? NCG : 1];
  int qk_pad[QKV ? NCG : 1];

  __device__ __forceinline__ void init(const GemmProb& P, int nw0, int mfirst, bool vcols, int lane) {
    const bf16_t* __restrict__ bias = (const bf16_t*)P.bias;
    const int N = P.N;
    // Reciprocals for div_exact, computed once: a division written in the
    // per-group code is expanded in full for every unrolled copy.
    inv_rpb = 1.0f / (float)P.rows_per_batch;
    if (QKV && !vcols) {
      const int D = P.hidden, dh = P.head_dim;
      const float inv_dh = 1.0f / (float)dh;
#pragma unroll
      for (int q = 0; q < NCG; ++q) {
        const int n = min(nw0 + ((lane + 64 * q) % CPR) * 4, N - 4);  // clamped: ragged strips
        const int sel = n >= D ? 1 : 0, rem = n - sel * D;  // q or k (v tiles take the other path)
        const int h = div_exact(rem, dh, inv_dh), d = rem - h * dh;
        qk_col[q] = (bf16_t*)(sel == 0 ? P.q : P.k) + (long)h * P.Tj * P.qk_stride + d;
        qk_f[q] = sel == 0 ? 1.0f : P.k_scale;  // k in the softmax's exp2 domain, rounded once
        qk_pad[q] = d + 4 == dh && P.qk_stride > dh ? 1 + sel : 0;
      }
    }
    if (EPI == EPI_QKV && vcols) {
#pragma unroll
      for (int it = 0; it < PL; ++it) {
        const int n = nw0 + (lane >> 3) + 8 * it;
        vb[it] = n < N ? bf2f(bias[n]) : 0.f;
      }
    }
    if (RES) {
      const int rpb = P.rows_per_batch;
      b0 = div_exact(min(mfirst, P.M - 1), rpb, inv_rpb);
    }
#pragma unroll
    for (int q = 0; q < NCG; ++q) {
      const int n = nw0 + ((lane + 64 * q) % CPR) * 4;  // N is a multiple of 4
      const u32x2 w = n < N ? *(const u32x2*)(bias + n) : u32x2{0u, 0u};
      bias4[q] = f32x4{__uint_as_float(w[0] << 16), __uint_as_float(w[0] & 0xFFFF0000u),
                       __uint_as_float(w[1] << 16), __uint_as_float(w[1] & 0xFFFF0000u)};
      if (RES)
        gate4[q] = n < N ? *(const f32x4*)(P.gate + (long)b0 * P.gate_stride + n) : f32x4{0.f, 0.f, 0.f, 0.f};
    }
  }

  // Residual rows of the slab at global row mb (EPI_RESID only).
  __device__ __forceinline__ void load_resid(f32x4 (&x)[NX], const GemmProb& P, int mb, int nw0, int lane) const {
    if (!RES || P.ksplit > 1) return;  // a split unit stores a raw partial
#pragma unroll
    for (int it = 0; it < PL; ++it) {
      const int c = lane + 64 * it;
      const int m = mb + c / CPR, n = nw0 + (c % CPR) * 4;
      x[it] = m < P.M && n < P.N ? *(const f32x4*)(P.resid + (long)m * P.N + n) : f32x4{0.f, 0.f, 0.f, 0.f};
    }
  }

  __device__ __forceinline__ void apply(const GemmProb& P, const float* Cw, int mb, int nw0, bool vcols, int lane,
                                        const f32x4 (&x)[NX]) const {
    const int rpb = P.rows_per_batch, M = P.M, N = P.N;
    if (EPI == EPI_QKV && vcols) {
      // v^T[b][h][d][j]: lane takes one column and four consecutive rows.
      // Element ((b H + h) dh + d) Tj_pad + v_key_pos(j), and h dh + d is the
      // column's offset n - 2D within the v block, so a lane's four rows
      // (fixed for the slab) give one row base and each column adds n Tj_pad.
      const int D = P.hidden;
      float cv[PL][4];  // all LDS reads first: one wait for the slab, not one per group
#pragma unroll
      for (int it = 0; it < PL; ++it) {
        const int c = lane + 64 * it;
        const int col = c >> 3, r4 = (c & 7) * 4;
#pragma unroll
        for (int e = 0; e < 4; ++e) cv[it][e] = Cw[(r4 + e) * CST + col];
      }
      const int m = mb + (lane & 7) * 4;  // the lane's first row: (c & 7) == (lane & 7)
      if (m >= M) return;
      const int b = div_exact(m, rpb, inv_rpb), j = m - b * rpb;
      const int jp = j + P.seq_off;
      const bool four = m + 3 < M && j + 3 < rpb && (jp & 3) == 0;  // 4 keys stay contiguous under v_key_pos
      bf16_t* const vrow = (bf16_t*)P.v + ((long)b * D - 2 * D) * P.Tj_pad + v_key_pos(jp);
#pragma unroll
      for (int it = 0; it < PL; ++it) {
        const int n = nw0 + ((lane + 64 * it) >> 3);
        if (n >= N) continue;
        const float bv = vb[it];
        const float v0 = cv[it][0] + bv, v1 = cv[it][1] + bv, v2 = cv[it][2] + bv, v3 = cv[it][3] + bv;
        if (four) {
          *(u32x2*)(vrow + (long)n * P.Tj_pad) = u32x2{pack_bf16x2(v0, v1), pack_bf16x2(v2, v3)};
        } else {
          const float vv[4] = {v0, v1, v2, v3};
          for (int e = 0; e < 4 && m + e < M; ++e) {
            const int be = div_exact(m + e, rpb, inv_rpb), je = (m + e) - be * rpb + P.seq_off;
            ((bf16_t*)P.v)[((long)be * D + n - 2 * D) * P.Tj_pad + v_key_pos(je)] = f2bf(vv[e]);
          }
        }
      }
      return;
    }
    f32x4 cy[PL];  // all LDS reads first: one wait for the slab, not one per group
#pragma unroll
    for (int it = 0; it < PL; ++it) {
      const int c = lane + 64 * it;
      cy[it] = *(const f32x4*)&Cw[(c / CPR) * CST + (c % CPR) * 4];
    }
    // Group it of the lane: row m, column n, element m N + n.  b: the row's
    // sample where it is known (-1: find it).
    auto group = [&](int it, int m, int n, long off, int b) __attribute__((always_inline)) {
      const f32x4 y = cy[it];
      if ((RES || EPI == EPI_GELU) && P.ksplit > 1) {  // one k-range: raw fp32 partial (P.part at its range)
        *(f32x4*)(P.part + off) = y;
        return;
      }
      const f32x4 bq = bias4[it % NCG];
      const float y0 = y[0] + bq[0], y1 = y[1] + bq[1], y2 = y[2] + bq[2], y3 = y[3] + bq[3];
      if (RES) {
        if (b < 0) b = div_exact(m, rpb, inv_rpb);
        f32x4 g = gate4[it % NCG];
        if (b != b0) g = *(const f32x4*)(P.gate + (long)b * P.gate_stride + n);  // strip spans two samples
        f32x4 xv = x[it];
        xv[0] += g[0] * y0;
        xv[1] += g[1] * y1;
        xv[2] += g[2] * y2;
        xv[3] += g[3] * y3;
        *(f32x4*)(P.resid + off) = xv;
      } else if (EPI == EPI_GELU) {
        *(u32x2*)((bf16_t*)P.out + off) =
            u32x2{pack_bf16x2(gelu_tanh(y0), gelu_tanh(y1)), pack_bf16x2(gelu_tanh(y2), gelu_tanh(y3))};
      } else if (EPI == EPI_STORE) {
        *(f32x4*)((float*)P.out + off) = f32x4{y0, y1, y2, y3};
      } else {  // EPI_QKV, q and k columns: 4 consecutive d of one head
        if (b < 0) b = div_exact(m, rpb, inv_rpb);
        const int jp = m - b * rpb + P.seq_off;
        bf16_t* dst = qk_col[it % NCG] + ((long)b * P.heads * P.Tj + jp) * P.qk_stride;
        const float f = qk_f[it % NCG];
        *(u32x2*)dst = u32x2{pack_bf16x2(y0 * f, y1 * f), pack_bf16x2(y2 * f, y3 * f)};
        // The row's padding (head_dim 72 -> 80) is zero, except k's column
        // head_dim, which is 1: there the attention kernel folds the running
        // softmax max into the QK^T product.
        if (qk_pad[it % NCG])
          for (int z = 4; z < P.qk_stride - P.head_dim + 4; z += 4)
            *(u32x2*)(dst + z) = u32x2{qk_pad[it % NCG] == 2 && z == 4 ? 0x3F80u : 0u, 0u};
      }
    };
    // A slab inside the matrix whose 32 rows belong to one sample (a lane's
    // column is the same in every group when CPR divides 64): no bounds
    // checks, one sample, and the row advances by 64 / CPR per group.
    bool fast = NCG == 1 && mb + 32 <= M && nw0 + WTN <= N;
    int bs = -1;
    if (fast && (RES || EPI == EPI_QKV)) {
      bs = div_exact(mb, rpb, inv_rpb);
      fast = div_exact(mb + 31, rpb, inv_rpb) == bs;
    }
    if (fast) {
      const int m = mb + lane / CPR, n = nw0 + (lane % CPR) * 4;
      const long off = (long)m * N + n;
#pragma unroll
      for (int it = 0; it < PL; ++it) group(it, m + (64 / CPR) * it, n, off + (long)((64 / CPR) * it) * N, bs);
      return;
    }
#pragma unroll
    for (int it = 0; it < PL; ++it) {
      const int c = lane + 64 * it;
      const int m = mb + c / CPR, n = nw0 + (c % CPR) * 4;
      if (m >= M || n >= N) continue;  // N is a multiple of 4
      group(it, m, n, (long)m * N + n, -1);
    }
  }
};

// Tile `local` of problem P -> its first row and column.  Tiles are taken in
// groups of P.group_m M-tiles x all N-tiles, M fastest within a group, so
// that consecutive tiles share W columns and a group's A rows stay in one
// L2; the XCDs run contiguous ranges of this order, and the host picks the
// group height that makes the range an XCD runs at once touch the fewest
// rows of A and W.
template <int BM, int BN>
__device__ __forceinline__ void tile_origin(const GemmProb& P, int local, int& m0, int& n0) {
  const int GM = max(P.group_m, 1);
  const int group_size = GM * P.tiles_n;
  const int group = local / group_size;
  const int first_m = group * GM;
  const int gm = min(P.tiles_m - first_m, GM);
  const int in_group = local - group * group_size;
  m0 = (first_m + in_group % gm) * BM;
  n0 = (in_group / gm) * BN;
}

// Main loop of one tile over the k-slices kb .. kb+nks-1 (nks >= 1) into acc,
// which it zeroes first.  On return every wave's DMA has landed and its LDS
// reads of the ring are complete, but other waves may still be reading: a
// workgroup barrier must precede any reuse of the LDS.
template <int BM, int BN, int WGM, int WGN, int STAGES>
__device__ __forceinline__ void gemm_mainloop(const GemmProb& P, int m0, int n0, int kb, int nks,
                                              f32x16 (&acc)[BM / WGM / 32][BN / WGN / 32],
                                              unsigned char* smem, unsigned lds0, int wave, int lane) {
  using C = GemmCfg<BM, BN, WGM, WGN, STAGES>;
  const bf16_t* __restrict__ A = (const bf16_t*)P.A + (long)kb * C::BK;
  const bf16_t* __restrict__ W = (const bf16_t*)P.W + (long)kb * C::BK;
  const int M = P.M, N = P.N, K = P.K;
  const int KT = nks;
  const int wm = wave / WGN, wn = wave - wm * WGN;
  const int r32 = lane & 31, g = lane >> 5;

  // DMA instruction t of this wave fills slice rows 8q .. 8q+7, q = wave + NW t;
  // lane -> row 8q + lane/8 at stored position lane%8, which holds chunk
  // (lane%8) ^ f(row) = (lane%8) ^ (lane/8) ^ (q&1), and q&1 = wave&1 (NW even).
  const int cfetch = (lane & 7) ^ (lane >> 3) ^ (wave & 1);
  unsigned voff[C::IPW];
#pragma unroll
  for (int t = 0; t < C::IPW; ++t) {
    const int row = 8 * (wave + C::NW * t) + (lane >> 3);
    const int grow = t < C::IPW_A ? min(m0 + row, M - 1) : min(n0 + row - BM, N - 1);  // clamped: ragged tiles
    voff[t] = (unsigned)grow * (unsigned)K * 2u + (unsigned)cfetch * 16u;
  }
  // DMA instruction t (0 <= t < IPW) of this wave for a slice into a slot.
  auto dma_one = [&](int slice, int slot, int t) {
    const bf16_t* src = (t < C::IPW_A ? A : W) + (long)slice * C::BK;
    dma_16s(src, voff[t], lds0 + (unsigned)(slot * C::SLICE + wave * 1024 + t * C::NW * 1024));
  };
  auto issue = [&](int slice, int slot) {
#pragma unroll
    for (int t = 0; t < C::IPW; ++t) dma_one(slice, slot, t);
  };

  // LDS read offsets of this lane's fragments within a slice buffer, per k-step s.
  int a_off[4][C::TM], b_off[4][C::TN];
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const int c = s * 2 + g;
#pragma unroll
    for (int i = 0; i < C::TM; ++i) {
      const int R = wm * C::WTM + i * 32 + r32;
      a_off[s][i] = R * 128 + (chunk_pos(R, c) << 4);
    }
#pragma unroll
    for (int j = 0; j < C::TN; ++j) {
      const int R = BM + wn * C::WTN + j * 32 + r32;
      b_off[s][j] = R * 128 + (chunk_pos(R, c) << 4);
    }
  }

#pragma unroll
  for (int i = 0; i < C::TM; ++i)
#pragma unroll
    for (int j = 0; j < C::TN; ++j) acc[i][j] = f32x16{};

#define GEMM_READ(FA, FB, slot, s)                                                            \
  do {                                                                                       \
    const unsigned char* b_ = smem + (slot) * C::SLICE;                                      \
    _Pragma("unroll") for (int i = 0; i < C::TM; ++i) FA[i] = *(const bf16x8*)(b_ + a_off[s][i]); \
    _Pragma("unroll") for (int j = 0; j < C::TN; ++j) FB[j] = *(const bf16x8*)(b_ + b_off[s][j]); \
  } while (0)
#define GEMM_MFMA(FA, FB)                                                                     \
  _Pragma("unroll") for (int i = 0; i < C::TM; ++i) _Pragma("unroll") for (int j = 0; j < C::TN; ++j) \
    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(FA[i], FB[j], acc[i][j], 0, 0, 0);
#define SCHED_FENCE() __builtin_amdgcn_sched_barrier(0)
  // One k-step's MFMAs with DMA instructions T0 .. T0+ND-1 of slice DSL
  // (into slot DSLOT) placed one after each MFMA, so the wave never waits for
  // the address unit with an MFMA still to issue.
#define GEMM_MFMA_DMA(FA, FB, ON, DSL, DSLOT, T0, ND)                                         \
  do {                                                                                       \
    _Pragma("unroll") for (int q = 0; q < C::TM * C::TN; ++q) {                              \
      acc[q / C::TN][q % C::TN] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(                   \
          FA[q / C::TN], FB[q % C::TN], acc[q / C::TN][q % C::TN], 0, 0, 0);                 \
      if (q < (ND)) {                                                                        \
        SCHED_FENCE();                                                                       \
        if (ON) dma_one(DSL, DSLOT, (T0) + q);                                               \
        SCHED_FENCE();                                                                       \
      }                                                                                      \
    }                                                                                        \
    _Pragma("unroll") for (int q = C::TM * C::TN; q < (ND); ++q) if (ON) dma_one(DSL, DSLOT, (T0) + q); \
  } while (0)

  // Slices past the end are not issued; where fewer than the steady-state
  // number are in flight, the waits fall back to vmcnt(0).
#pragma unroll
  for (int s = 0; s < STAGES; ++s)
    if (s < KT) issue(s, s);
  if (KT >= STAGES) wait_vmcnt<(STAGES - 1) * C::IPW>();
  else wait_vmcnt<0>();
  __syncthreads();

  // Software pipeline over slices (4 MFMA k-steps each), fragments double
  // buffered per k-step in X (even k-steps) and Y (odd).  Entering iteration
  // kt, X holds k-step 0 of slice kt.  Each k-step's reads are issued before
  // the previous k-step's MFMAs.  After the last reads of slot kt, the wave
  // waits for its DMA of slice kt+1; the workgroup barrier then guarantees
  // every wave's DMA of kt+1 has landed and every read of slot kt is
  // complete, so slice kt+STAGES may be written into that slot.  Its DMA
  // instructions are spread over two MFMA groups (the last k-step of slice kt
  // and the first of slice kt+1): issued as one burst, the whole workgroup's
  // DMA queues behind the address unit (16 cycles per 1 KB instruction) and
  // the waves stall at issue with their MFMAs still to go.
  constexpr int H1 = C::IPW / 2, H2 = C::IPW - H1;
  bf16x8 xa[C::TM], xb[C::TN], ya[C::TM], yb[C::TN];
  GEMM_READ(xa, xb, 0, 0);
  int slot = 0;
  // One slice.  dma1 / dma2: whether the two refills (slices kt-1+STAGES and
  // kt+STAGES) exist, mid: both exist and slice kt+1 is not the last in
  // flight.  The loop below runs the slices where all three hold with
  // literal true, so the steady state has no branches around its DMAs.
  auto iteration = [&](const int kt, const bool dma1, const bool dma2, const bool mid) __attribute__((always_inline)) {
    const int next = slot + 1 == STAGES ? 0 : slot + 1;
    const int prev = slot == 0 ? STAGES - 1 : slot - 1;  // slot of slice kt-1, refilled with kt-1+STAGES
    GEMM_READ(ya, yb, slot, 1);
    SCHED_FENCE();
    GEMM_MFMA_DMA(xa, xb, dma1, kt - 1 + STAGES, prev, H1, H2);
    SCHED_FENCE();
    GEMM_READ(xa, xb, slot, 2);
    SCHED_FENCE();
    GEMM_MFMA(ya, yb);
    SCHED_FENCE();
    GEMM_READ(ya, yb, slot, 3);
    SCHED_FENCE();
    GEMM_MFMA(xa, xb);
    SCHED_FENCE();
    if (mid) wait_vmcnt<(STAGES - 2) * C::IPW>();  // own DMA of slice kt+1 landed
    else wait_vmcnt<0>();
    __syncthreads();
    GEMM_READ(xa, xb, next, 0);  // past the last slice this reads stale data, unused
    SCHED_FENCE();
    GEMM_MFMA_DMA(ya, yb, dma2, kt + STAGES, slot, 0, H1);
    SCHED_FENCE();
    slot = next;
  };
  auto generic = [&](const int kt) __attribute__((always_inline)) {
    iteration(kt, kt >= 1 && kt - 1 + STAGES < KT, kt + STAGES < KT, kt + STAGES - 1 < KT);
  };
  // slices 1 .. KT-STAGES-1 have both refills and a slice in flight behind kt+1
  const int steady_end = KT - STAGES;
  if (KT > 0) generic(0);
  int kt = 1;
  for (; kt < steady_end; ++kt) iteration(kt, true, true, true);
  for (; kt < KT; ++kt) generic(kt);
#undef GEMM_READ
#undef GEMM_MFMA
#undef GEMM_MFMA_DMA
#undef SCHED_FENCE
}

// Epilogue of one tile from the accumulators.  Per 32-row slab i: each wave
// writes its 32 x WTN accumulators to its own LDS region (column r32 + 32j,
// rows 8*jj + 4*g + ii), then reads them back four columns (or, for v^T,
// four rows) per lane.  The residual rows of slab i+1 are requested before
// slab i is processed.  A wave only reads back its own LDS region, and the
// LDS executes one wave's instructions in order, so after one workgroup
// barrier (every wave is done with the slice ring, which the regions
// overlap) the slabs need no further barriers, only a wavefront-scope fence
// that keeps the compiler from reordering the lanes' LDS writes and reads.
template <int BM, int BN, int WGM, int WGN, int STAGES, int EPI>
__device__ __forceinline__ void gemm_epilogue(const GemmProb& P, int m0, int n0, bool vcols,
                                              const Epilogue<EPI, BN / WGN, BN / WGN + 4>& epi,
                                              const f32x16 (&acc)[BM / WGM / 32][BN / WGN / 32],
                                              unsigned char* smem, int wave, int lane) {
  using C = GemmCfg<BM, BN, WGM, WGN, STAGES>;
  using E = Epilogue<EPI, C::WTN, C::CST>;
  const int wm = wave / WGN, wn = wave - wm * WGN;
  const int r32 = lane & 31, g = lane >> 5;
  float* const Cw = reinterpret_cast<float*>(smem) + wave * 32 * C::CST;
  const int mw0 = m0 + wm * C::WTM, nw0 = n0 + wn * C::WTN;
  f32x4 xcur[E::NX], xnext[E::NX];
  epi.load_resid(xcur, P, mw0, nw0, lane);
  __syncthreads();
#pragma unroll
  for (int i = 0; i < C::TM; ++i) {
    wave_lds_fence();
#pragma unroll
    for (int j = 0; j < C::TN; ++j)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
#pragma unroll
        for (int ii = 0; ii < 4; ++ii) Cw[(jj * 8 + g * 4 + ii) * C::CST + j * 32 + r32] = acc[i][j][jj * 4 + ii];
    wave_lds_fence();
    if (i + 1 < C::TM) epi.load_resid(xnext, P, mw0 + (i + 1) * 32, nw0, lane);
    epi.apply(P, Cw, mw0 + i * 32, nw0, vcols, lane, xcur);
#pragma unroll
    for (int t = 0; t < E::NX; ++t) xcur[t] = xnext[t];
  }
}

// One tile per workgroup.
template <int BM, int BN, int WGM, int WGN, int STAGES, int EPI>
__global__ __launch_bounds__(WGM * WGN * 64) void gemm_bf16_kernel(GemmArgs args) {
  using C = GemmCfg<BM, BN, WGM, WGN, STAGES>;
  __shared__ __attribute__((aligned(1024))) unsigned char smem[C::LDS];

  int tile;
  if (args.tail) {  // XCD x = blockIdx % 8 runs n0 tiles of problem 0, then n1 units of problem 1
    const int n0 = args.p[1].tile_begin >> 3, n1 = (args.total_tiles - args.p[1].tile_begin) >> 3;
    const int xcd = blockIdx.x & 7, idx = blockIdx.x >> 3;
    tile = idx < n0 ? xcd * n0 + idx : args.p[1].tile_begin + xcd * n1 + (idx - n0);
  } else {
    tile = xcd_remap(blockIdx.x, args.total_tiles);
  }
  // Select the problem by value: indexing the by-value argument array with a
  // runtime index would copy it to scratch memory.
  const bool second = args.nprob > 1 && tile >= args.p[1].tile_begin;
  GemmProb P = second ? args.p[1] : args.p[0];
  // Split K: unit u of the problem is k-range u / (tiles_m tiles_n) of tile
  // u % (tiles_m tiles_n).
  int local = tile - P.tile_begin, kb = 0, nks = P.K / C::BK;
  if ((EPI == EPI_GELU || EPI == EPI_RESID || EPI == EPI_RESID2) && P.ksplit > 1) {
    const int per = P.tiles_m * P.tiles_n, s = local / per;
    local -= s * per;
    nks /= P.ksplit;
    kb = s * nks;
    P.part += (long)s * P.M * P.N;
  }
  int m0, n0;
  tile_origin<BM, BN>(P, local, m0, n0);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (scalar) index
  const int wm = wave / WGN, wn = wave - wm * WGN;
  const unsigned lds0 = __builtin_amdgcn_readfirstlane(lds_address(smem));

  // Epilogue constants (bias, gate) are requested first, so they are resident
  // long before the epilogue; being older than every DMA, they never delay
  // the explicit vmcnt waits of the main loop.
  using E = Epilogue<EPI, C::WTN, C::CST>;
  const bool vcols = EPI == EPI_QKV && n0 >= 2 * P.hidden;  // tiles never straddle k|v (2D % BN == 0)
  E epi;
  epi.init(P, n0 + wn * C::WTN, m0 + wm * C::WTM, vcols, lane);

  f32x16 acc[C::TM][C::TN];
  gemm_mainloop<BM, BN, WGM, WGN, STAGES>(P, m0, n0, kb, nks, acc, smem, lds0, wave, lane);
  gemm_epilogue<BM, BN, WGM, WGN, STAGES, EPI>(P, m0, n0, vcols, epi, acc, smem, wave, lane);
}

// ---------------------------------------------------------------- 64 x 144 tiles
// For N a multiple of 144 (the DiT-XL widths 1152 = 8*144, 3456 = 24*144,
// 4608 = 32*144), 64 x 144 tiles make the tile count a multiple of 256 at the
// DiT-XL/2 token counts (2048 or 4096 rows), so every CU gets the same work;
// 64 x 128 or 128 x 128 tiles there leave part of the last round idle.
// Six waves (2 x 3), each owning 32 x 48 as 2 x 3 accumulators of
// v_mfma_f32_16x16x32_bf16 (lane: row lane%16 of A and of W, k offset
// 8*(lane/16) + 32*step; D: column lane%16, rows 4*(lane/16) + i).  Same
// slice format, swizzle, DMA ring and refill rule as the kernel above; the
// slice's 26 DMA instructions are spread 5 per wave, and the 4 spare ones
// re-read a valid row into a dummy LDS line.  Six waves leave two SIMDs with
// two waves and two with one, so with KG = 2 the workgroup holds two such
// k-groups of six waves (three waves per SIMD), each with its own ring of
// 3 x 26 KB, taking alternate k-slices; at the end k-group 1 hands its
// partial sums to k-group 0 through LDS.  With KG = 1 the ring lets two
// workgroups share a CU.
template <int KG>
struct Gemm144 {
  static constexpr int BM = 64, BN = 144, BK = 64, STAGES = 3, NW = 6;  // per k-group
  static constexpr int ROWS = BM + BN;                // 208
  static constexpr int SLICE = ROWS * 128;            // bytes per slice buffer
  static constexpr int NDMA = ROWS / 8;               // 26 DMA instructions per slice
  static constexpr int IPW = (NDMA + NW - 1) / NW;    // 5 per wave
  static constexpr int TM = 2, TN = 3, WTM = 32, WTN = 48;
  static constexpr int CST = WTN + 4;                 // fp32 row stride of an epilogue slab
  static constexpr int SPARE = KG * STAGES * SLICE;   // dummy target of the spare DMAs
  static constexpr int LDS_MAIN = SPARE + 1024;
  static constexpr int LDS_EPI = NW * 32 * CST * 4;
  static constexpr int LDS = LDS_MAIN > LDS_EPI ? LDS_MAIN : LDS_EPI;
  static_assert((STAGES - 1) * IPW < 64, "vmcnt range");
  static_assert(KG == 2 || 2 * LDS <= 160 * 1024, "two workgroups per CU");
  static_assert(LDS <= 160 * 1024, "LDS per CU");
  static_assert(TM * TN * 4 * 64 <= 32 * CST, "a k-group's partial fits the wave's epilogue region");
};

template <int EPI, int KG>
__global__ __launch_bounds__(384 * KG) void gemm_bf16_144_kernel(GemmArgs args) {
  using C = Gemm144<KG>;
  __shared__ __attribute__((aligned(1024))) unsigned char smem[C::LDS];

  const int tile = xcd_remap(blockIdx.x, args.total_tiles);
  const bool second = args.nprob > 1 && tile >= args.p[1].tile_begin;
  const GemmProb P = second ? args.p[1] : args.p[0];
  const int local = tile - P.tile_begin;
  const int GM = max(P.group_m, 1);  // as tile_origin
  const int group_size = GM * P.tiles_n;
  const int group = local / group_size;
  const int first_m = group * GM;
  const int gm = min(P.tiles_m - first_m, GM);
  const int in_group = local - group * group_size;
  const int m0 = (first_m + in_group % gm) * C::BM;
  const int n0 = (in_group / gm) * C::BN;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave_id = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int kg = wave_id / C::NW;                 // k-group: slices kg, kg + KG, kg + 2 KG, ...
  const int wave = wave_id - kg * C::NW;          // wave within the k-group
  const bf16_t* __restrict__ A = (const bf16_t*)P.A + kg * C::BK;
  const bf16_t* __restrict__ W = (const bf16_t*)P.W + kg * C::BK;
  const int M = P.M, N = P.N, K = P.K;
  const int KT = K / (C::BK * KG);                // slices per k-group (K / 64 is a multiple of KG)
  const int wm = wave / 3, wn = wave - 3 * wm;
  const int r16 = lane & 15, g4 = lane >> 4;
  const unsigned lds0 = __builtin_amdgcn_readfirstlane(lds_address(smem)) + (unsigned)(kg * C::STAGES * C::SLICE);

  // DMA instruction t of this wave fills slice rows 8q .. 8q+7, q = wave + 6t
  // (A rows for q < 8, W rows for q < 26, spare above); lane -> row 8q +
  // lane/8 at stored position lane%8, i.e. chunk (lane%8) ^ (lane/8) ^ (q&1).
  const int cfetch = (lane & 7) ^ (lane >> 3) ^ (wave & 1);
  unsigned voff[C::IPW];
#pragma unroll
  for (int t = 0; t < C::IPW; ++t) {
    const int q = wave + C::NW * t;
    const int row = 8 * q + (lane >> 3);
    const int grow = q < C::BM / 8 ? min(m0 + row, M - 1) : q < C::NDMA ? min(n0 + row - C::BM, N - 1) : 0;
    voff[t] = (unsigned)grow * (unsigned)K * 2u + (unsigned)cfetch * 16u;
  }
  auto dma_one = [&](int slice, int slot, int t) {
    const int q = wave + C::NW * t;  // wave-uniform
    const unsigned dst = q < C::NDMA ? lds0 + (unsigned)(slot * C::SLICE + q * 1024)
                                     : lds0 - (unsigned)(kg * C::STAGES * C::SLICE) + (unsigned)C::SPARE;
    dma_16s((q < C::BM / 8 || q >= C::NDMA ? A : W) + (long)slice * (KG * C::BK), voff[t], dst);
  };
  auto issue = [&](int slice, int slot) {
#pragma unroll
    for (int t = 0; t < C::IPW; ++t) dma_one(slice, slot, t);
  };

  // fragment offsets per 32-wide k-step s (two per slice)
  int a_off[2][C::TM], b_off[2][C::TN];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int c = 4 * s + g4;
#pragma unroll
    for (int i = 0; i < C::TM; ++i) {
      const int R = wm * C::WTM + i * 16 + r16;
      a_off[s][i] = R * 128 + (chunk_pos(R, c) << 4);
    }
#pragma unroll
    for (int j = 0; j < C::TN; ++j) {
      const int R = C::BM + wn * C::WTN + j * 16 + r16;
      b_off[s][j] = R * 128 + (chunk_pos(R, c) << 4);
    }
  }

  f32x4 acc[C::TM][C::TN];
#pragma unroll
  for (int i = 0; i < C::TM; ++i)
#pragma unroll
    for (int j = 0; j < C::TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  bf16x8 xa[C::TM], xb[C::TN], ya[C::TM], yb[C::TN];
#define G144_READ(FA, FB, slot, s)                                                            \
  do {                                                                                       \
    const unsigned char* b_ = smem + (kg * C::STAGES + (slot)) * C::SLICE;                   \
    _Pragma("unroll") for (int i = 0; i < C::TM; ++i) FA[i] = *(const bf16x8*)(b_ + a_off[s][i]); \
    _Pragma("unroll") for (int j = 0; j < C::TN; ++j) FB[j] = *(const bf16x8*)(b_ + b_off[s][j]); \
  } while (0)
#define G144_MFMA(FA, FB)                                                                     \
  _Pragma("unroll") for (int i = 0; i < C::TM; ++i) _Pragma("unroll") for (int j = 0; j < C::TN; ++j) \
    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(FA[i], FB[j], acc[i][j], 0, 0, 0);
#define SCHED_FENCE() __builtin_amdgcn_sched_barrier(0)
  // As in the kernel above: a slice's DMA instructions are placed between the
  // MFMAs of two k-steps instead of being issued as one burst.
#define G144_MFMA_DMA(FA, FB, ON, DSL, DSLOT, T0, ND)                                         \
  do {                                                                                       \
    _Pragma("unroll") for (int q = 0; q < C::TM * C::TN; ++q) {                              \
      acc[q / C::TN][q % C::TN] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(                   \
          FA[q / C::TN], FB[q % C::TN], acc[q / C::TN][q % C::TN], 0, 0, 0);                 \
      if (q < (ND)) {                                                                        \
        SCHED_FENCE();                                                                       \
        if (ON) dma_one(DSL, DSLOT, (T0) + q);                                               \
        SCHED_FENCE();                                                                       \
      }                                                                                      \
    }                                                                                        \
    _Pragma("unroll") for (int q = C::TM * C::TN; q < (ND); ++q) if (ON) dma_one(DSL, DSLOT, (T0) + q); \
  } while (0)

  using E = Epilogue<EPI, C::WTN, C::CST>;
  const int mw0 = m0 + wm * C::WTM, nw0 = n0 + wn * C::WTN;
  const bool vcols = EPI == EPI_QKV && n0 >= 2 * P.hidden;  // the host only picks 144 when 2D % 144 == 0
  E epi;
  if (kg == 0) epi.init(P, nw0, mw0, vcols, lane);

#pragma unroll
  for (int s = 0; s < C::STAGES; ++s)
    if (s < KT) issue(s, s);
  if (KT >= C::STAGES) wait_vmcnt<(C::STAGES - 1) * C::IPW>();
  else wait_vmcnt<0>();
  __syncthreads();
  constexpr int H1 = C::IPW / 2, H2 = C::IPW - H1;
  G144_READ(xa, xb, 0, 0);
  int slot = 0;
  for (int kt = 0; kt < KT; ++kt) {
    const int next = slot + 1 == C::STAGES ? 0 : slot + 1;
    const int prev = slot == 0 ? C::STAGES - 1 : slot - 1;  // slot of slice kt-1, refilled with kt-1+STAGES
    G144_READ(ya, yb, slot, 1);
    SCHED_FENCE();
    G144_MFMA_DMA(xa, xb, kt >= 1 && kt - 1 + C::STAGES < KT, kt - 1 + C::STAGES, prev, H1, H2);
    SCHED_FENCE();
    if (kt + C::STAGES - 1 < KT) wait_vmcnt<(C::STAGES - 2) * C::IPW>();  // own DMA of slice kt+1 landed
    else wait_vmcnt<0>();
    __syncthreads();
    G144_READ(xa, xb, next, 0);  // past the last slice this reads stale data, unused
    SCHED_FENCE();
    G144_MFMA_DMA(ya, yb, kt + C::STAGES < KT, kt + C::STAGES, slot, 0, H1);
    SCHED_FENCE();
    slot = next;
  }
#undef G144_READ
#undef G144_MFMA
#undef G144_MFMA_DMA
#undef SCHED_FENCE

  // epilogue: each wave stages its 32 x 48 accumulators in its own LDS region
  float* const Cw = reinterpret_cast<float*>(smem) + wave * 32 * C::CST;
  f32x4 xr[E::NX];
  if (kg == 0) epi.load_resid(xr, P, mw0, nw0, lane);
  __syncthreads();  // every wave is done with the slice ring
  if (KG == 2) {
    // k-group 1 hands its partial sums to the wave of k-group 0 that owns
    // the same outputs, through that wave's epilogue region (lane-major),
    // and leaves; that wave adds them before staging its own.
    if (kg == 1) {
#pragma unroll
      for (int i = 0; i < C::TM; ++i)
#pragma unroll
        for (int j = 0; j < C::TN; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e) Cw[((i * C::TN + j) * 4 + e) * 64 + lane] = acc[i][j][e];
    }
    __syncthreads();
    if (kg == 1) return;
#pragma unroll
    for (int i = 0; i < C::TM; ++i)
#pragma unroll
      for (int j = 0; j < C::TN; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[i][j][e] += Cw[((i * C::TN + j) * 4 + e) * 64 + lane];
    wave_lds_fence();  // the partial is read before the region is overwritten
  }
#pragma unroll
  for (int i = 0; i < C::TM; ++i)
#pragma unroll
    for (int j = 0; j < C::TN; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) Cw[(i * 16 + 4 * g4 + e) * C::CST + j * 16 + r16] = acc[i][j][e];
  wave_lds_fence();  // own region only: the LDS runs a wave's accesses in order
  epi.apply(P, Cw, mw0, nw0, vcols, lane, xr);
}

// Split-K reduction: four consecutive outputs per lane, 16-byte loads of
// each k-range's partial; bias, GELU and bf16 rounding as in the GEMM
// epilogue.
__global__ __launch_bounds__(256) void splitk_gelu_kernel(const float* __restrict__ part, int S, long MN, int N,
                                                          const bf16_t* __restrict__ bias, bf16_t* __restrict__ out) {
  const long e = (blockIdx.x * 256L + threadIdx.x) * 4;
  if (e >= MN) return;
  f32x4 y = *(const f32x4*)(part + e);
  for (int s = 1; s < S; ++s) {
    const f32x4 p = *(const f32x4*)(part + s * MN + e);
    y[0] += p[0];
    y[1] += p[1];
    y[2] += p[2];
    y[3] += p[3];
  }
  const int n = (int)(e % N);
  const u32x2 w = *(const u32x2*)(bias + n);
  const float y0 = y[0] + __uint_as_float(w[0] << 16), y1 = y[1] + __uint_as_float(w[0] & 0xFFFF0000u);
  const float y2 = y[2] + __uint_as_float(w[1] << 16), y3 = y[3] + __uint_as_float(w[1] & 0xFFFF0000u);
  *(u32x2*)(out + e) = u32x2{pack_bf16x2(gelu_tanh(y0), gelu_tanh(y1)), pack_bf16x2(gelu_tanh(y2), gelu_tanh(y3))};
}

hipError_t launch_splitk_gelu_bf16(const float* part, int S, int M, int N, const void* bias, void* out,
                                   hipStream_t st) {
  const long MN = (long)M * N;
  if (MN == 0) return hipSuccess;
  const long groups = MN / 4;
  hipLaunchKernelGGL(splitk_gelu_kernel, dim3((unsigned)((groups + 255) / 256)), dim3(256), 0, st, part, S, MN, N,
                     (const bf16_t*)bias, (bf16_t*)out);
  return hipGetLastError();
}

// Split-K reduction into the fp32 residual: four consecutive outputs per
// lane; the ranges are added in order, then the bias, then the gated update
// as in the GEMM's residual epilogue.
__global__ __launch_bounds__(256) void splitk_resid_kernel(const float* __restrict__ part, int S, long MN, int N,
                                                           const bf16_t* __restrict__ bias,
                                                           const float* __restrict__ gate, int gate_stride,
                                                           int rows_per_batch, float* __restrict__ resid) {
  const long e = (blockIdx.x * 256L + threadIdx.x) * 4;
  if (e >= MN) return;
  f32x4 y = *(const f32x4*)(part + e);
  for (int s = 1; s < S; ++s) {
    const f32x4 p = *(const f32x4*)(part + s * MN + e);
    y[0] += p[0];
    y[1] += p[1];
    y[2] += p[2];
    y[3] += p[3];
  }
  const long m = e / N;
  const int n = (int)(e - m * N), b = (int)(m / rows_per_batch);
  const u32x2 w = *(const u32x2*)(bias + n);
  const f32x4 g = *(const f32x4*)(gate + (long)b * gate_stride + n);
  f32x4 x = *(const f32x4*)(resid + e);
  x[0] += g[0] * (y[0] + __uint_as_float(w[0] << 16));
  x[1] += g[1] * (y[1] + __uint_as_float(w[0] & 0xFFFF0000u));
  x[2] += g[2] * (y[2] + __uint_as_float(w[1] << 16));
  x[3] += g[3] * (y[3] + __uint_as_float(w[1] & 0xFFFF0000u));
  *(f32x4*)(resid + e) = x;
}

hipError_t launch_splitk_resid(const float* part, int S, int M, int N, const void* bias, const float* gate,
                               int gate_stride, int rows_per_batch, float* resid, hipStream_t st) {
  const long MN = (long)M * N;
  if (MN == 0) return hipSuccess;
  hipLaunchKernelGGL(splitk_resid_kernel, dim3((unsigned)((MN / 4 + 255) / 256)), dim3(256), 0, st, part, S, MN, N,
                     (const bf16_t*)bias, gate, gate_stride, rows_per_batch, resid);
  return hipGetLastError();
}

void gemm_tile_dims(int tile_cfg, int* bm, int* bn) {
  switch (tile_cfg) {
    case TILE_128x128: *bm = 128; *bn = 128; break;
    case TILE_64x144:
    case TILE_64x144_1: *bm = 64; *bn = 144; break;
    case TILE_256x256: *bm = 256; *bn = 256; break;
    case TILE_256x128: *bm = 256; *bn = 128; break;
    case TILE_256x192: *bm = 256; *bn = 192; break;
    default: *bm = 64; *bn = 128; break;
  }
}

template <int KG>
static hipError_t launch_144_kg(const GemmArgs& a, int epi, hipStream_t st) {
  dim3 grid(a.total_tiles), block(Gemm144<KG>::NW * KG * 64);
  switch (epi) {
    case EPI_QKV: hipLaunchKernelGGL((gemm_bf16_144_kernel<EPI_QKV, KG>), grid, block, 0, st, a); break;
    case EPI_GELU: hipLaunchKernelGGL((gemm_bf16_144_kernel<EPI_GELU, KG>), grid, block, 0, st, a); break;
    case EPI_RESID: hipLaunchKernelGGL((gemm_bf16_144_kernel<EPI_RESID, KG>), grid, block, 0, st, a); break;
    case EPI_RESID2: hipLaunchKernelGGL((gemm_bf16_144_kernel<EPI_RESID2, KG>), grid, block, 0, st, a); break;
    default: hipLaunchKernelGGL((gemm_bf16_144_kernel<EPI_STORE, KG>), grid, block, 0, st, a); break;
  }
  return hipGetLastError();
}

// Two k-groups (twelve waves, three per SIMD) where every problem has an
// even number of k-slices; one group of six waves otherwise.
static hipError_t launch_144(const GemmArgs& a, int epi, hipStream_t st) {
  bool even = true;
  for (int i = 0; i < a.nprob; ++i) even = even && (a.p[i].K / 64) % 2 == 0;
  return even ? launch_144_kg<2>(a, epi, st) : launch_144_kg<1>(a, epi, st);
}

template <int BM, int BN, int WGM, int WGN, int STAGES>
static hipError_t launch_tile(const GemmArgs& a, int epi, hipStream_t st) {
  dim3 grid(a.total_tiles), block(WGM * WGN * 64);
#define GEMM_EPI_CASE(E) hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, WGM, WGN, STAGES, E>), grid, block, 0, st, a)
  switch (epi) {
    case EPI_QKV: GEMM_EPI_CASE(EPI_QKV); break;
    case EPI_GELU: GEMM_EPI_CASE(EPI_GELU); break;
    case EPI_RESID: GEMM_EPI_CASE(EPI_RESID); break;
    case EPI_RESID2: GEMM_EPI_CASE(EPI_RESID2); break;
    default: GEMM_EPI_CASE(EPI_STORE); break;
  }
#undef GEMM_EPI_CASE
  return hipGetLastError();
}

// Ring depth: a slice is (BM + BN) x 128 bytes, so 128x128 with 2 slots and
// 64x128 with 3 fit two workgroups per CU (64 KB, 72 KB), and 64x128 with 2
// slots fits three (48 KB); measured faster than deeper rings with one
// workgroup per CU.  256x256 (2 slots, 128 KB) and 256x128 (3 slots, 144 KB)
// run one eight-wave workgroup per CU.
hipError_t launch_gemm_bf16(const GemmArgs& a, int epi, int tile_cfg, hipStream_t st) {
  switch (tile_cfg) {
    case TILE_64x128: return launch_tile<64, 128, 2, 2, 3>(a, epi, st);
    case TILE_64x128_S2: return launch_tile<64, 128, 2, 2, 2>(a, epi, st);
    case TILE_64x144: return launch_144(a, epi, st);
    case TILE_64x144_1: return launch_144_kg<1>(a, epi, st);
    case TILE_256x256: return launch_tile<256, 256, 2, 4, 2>(a, epi, st);
    case TILE_256x128: return launch_tile<256, 128, 4, 2, 3>(a, epi, st);
    case TILE_256x192: return launch_tile<256, 192, 4, 2, 2>(a, epi, st);
    default: return launch_tile<128, 128, 2, 2, 2>(a, epi, st);
  }
}

}  // namespace ditmi
