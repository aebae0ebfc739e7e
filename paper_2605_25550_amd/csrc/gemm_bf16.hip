// bf16 MFMA GEMM for the DiT block's linear layers (QKV, output projection,
// MLP fc1/fc2 and the final layer) on gfx950:
//   y[M, N] = A[M, K] * W[N, K]^T + bias,  fp32 accumulate,
// followed by a fused epilogue (kernels.h: Epi).  Both operands are
// K-contiguous, so every lane of a v_mfma_f32_32x32x16_bf16 reads 8
// consecutive bf16 (16 bytes) of one row from LDS.
//
// Tiling: BM x BN x 64 per workgroup of 4 waves (2 x 2), each wave owns a
// (BM/2) x (BN/2) sub-tile of 32x32 accumulators.  Global -> VGPR -> LDS
// staging with two LDS buffers: the next K slice is fetched from HBM while
// the current one feeds the matrix cores; one barrier per K slice.  LDS rows
// carry 16 bytes of padding so the 32 rows read by a half-wavefront hit
// distinct banks.  Workgroup ids are remapped so that neighbouring tiles
// (which share A rows) run on the same XCD and its L2.
#include "common.h"
#include "kernels.h"

namespace ditmi {

template <int BM, int BN>
struct GemmCfg {
  static constexpr int BK = 64;
  static constexpr int LDK = BK + 8;  // bf16 per LDS row
  static constexpr int WTM = BM / 2, WTN = BN / 2;
  static constexpr int TM = WTM / 32, TN = WTN / 32;
  static constexpr int A_CH = BM * BK / 8 / 256;  // 16-byte chunks per thread
  static constexpr int B_CH = BN * BK / 8 / 256;
};

template <int BM, int BN, int EPI>
__global__ __launch_bounds__(256) void gemm_bf16_kernel(GemmArgs args) {
  using C = GemmCfg<BM, BN>;
  __shared__ __attribute__((aligned(16))) bf16_t As[2][BM * C::LDK];
  __shared__ __attribute__((aligned(16))) bf16_t Bs[2][BN * C::LDK];

  const int tile = xcd_remap(blockIdx.x, args.total_tiles);
  // Select the problem field by field: indexing the by-value argument array
  // with a runtime index would copy it to scratch memory.
  const bool second = args.nprob > 1 && tile >= args.p[1].tile_begin;
  const GemmProb P = second ? args.p[1] : args.p[0];
  const int local = tile - P.tile_begin;
  const int GM = 8;
  const int group_size = GM * P.tiles_n;
  const int group = local / group_size;
  const int first_m = group * GM;
  const int gm = min(P.tiles_m - first_m, GM);
  const int in_group = local - group * group_size;
  const int m0 = (first_m + in_group % gm) * BM;
  const int n0 = (in_group / gm) * BN;

  const bf16_t* __restrict__ A = (const bf16_t*)P.A;
  const bf16_t* __restrict__ W = (const bf16_t*)P.W;
  const int M = P.M, N = P.N, K = P.K;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int r32 = lane & 31, g = lane >> 5;

  const bf16_t* a_src[C::A_CH];
  int a_dst[C::A_CH];
#pragma unroll
  for (int i = 0; i < C::A_CH; ++i) {
    int c = tid + 256 * i, row = c >> 3, kc = c & 7;
    int grow = min(m0 + row, M - 1);
    a_src[i] = A + (long)grow * K + kc * 8;
    a_dst[i] = row * C::LDK + kc * 8;
  }
  const bf16_t* b_src[C::B_CH];
  int b_dst[C::B_CH];
#pragma unroll
  for (int i = 0; i < C::B_CH; ++i) {
    int c = tid + 256 * i, row = c >> 3, kc = c & 7;
    int grow = min(n0 + row, N - 1);
    b_src[i] = W + (long)grow * K + kc * 8;
    b_dst[i] = row * C::LDK + kc * 8;
  }

  uint4 ra[C::A_CH], rb[C::B_CH];
#define GEMM_GLOAD(k0)                                                                \
  do {                                                                               \
    _Pragma("unroll") for (int i = 0; i < C::A_CH; ++i) ra[i] = *(const uint4*)(a_src[i] + (k0)); \
    _Pragma("unroll") for (int i = 0; i < C::B_CH; ++i) rb[i] = *(const uint4*)(b_src[i] + (k0)); \
  } while (0)
#define GEMM_LSTORE(buf)                                                              \
  do {                                                                               \
    _Pragma("unroll") for (int i = 0; i < C::A_CH; ++i) *(uint4*)&As[buf][a_dst[i]] = ra[i]; \
    _Pragma("unroll") for (int i = 0; i < C::B_CH; ++i) *(uint4*)&Bs[buf][b_dst[i]] = rb[i]; \
  } while (0)

  f32x16 acc[C::TM][C::TN];
#pragma unroll
  for (int i = 0; i < C::TM; ++i)
#pragma unroll
    for (int j = 0; j < C::TN; ++j) acc[i][j] = f32x16{};

#define GEMM_COMPUTE(buf)                                                                            \
  do {                                                                                              \
    _Pragma("unroll") for (int kk = 0; kk < C::BK / 16; ++kk) {                                     \
      bf16x8 af[C::TM], bw[C::TN];                                                                  \
      _Pragma("unroll") for (int i = 0; i < C::TM; ++i)                                             \
        af[i] = *(const bf16x8*)&As[buf][(wm * C::WTM + i * 32 + r32) * C::LDK + kk * 16 + g * 8];  \
      _Pragma("unroll") for (int j = 0; j < C::TN; ++j)                                             \
        bw[j] = *(const bf16x8*)&Bs[buf][(wn * C::WTN + j * 32 + r32) * C::LDK + kk * 16 + g * 8];  \
      _Pragma("unroll") for (int i = 0; i < C::TM; ++i)                                             \
        _Pragma("unroll") for (int j = 0; j < C::TN; ++j)                                           \
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bw[j], acc[i][j], 0, 0, 0);    \
    }                                                                                               \
  } while (0)

  // The last K slice is peeled so the prefetch in the steady-state loop is
  // unconditional (a conditional prefetch makes the compiler keep the staging
  // registers in scratch memory).
  const int KT = K / C::BK;
  GEMM_GLOAD(0);
  GEMM_LSTORE(0);
  __syncthreads();
  for (int kt = 0; kt + 1 < KT; ++kt) {
    const int buf = kt & 1;
    GEMM_GLOAD((kt + 1) * C::BK);
    GEMM_COMPUTE(buf);
    GEMM_LSTORE(buf ^ 1);
    __syncthreads();
  }
  GEMM_COMPUTE((KT - 1) & 1);
#undef GEMM_COMPUTE
#undef GEMM_GLOAD
#undef GEMM_LSTORE

  // ---------------------------------------------------------------- epilogue
  // Lane holds column n = (wave col) + j*32 + r32 and rows 8*jj + 4*g + ii.
  const bf16_t* __restrict__ bias = (const bf16_t*)P.bias;
  float bn[C::TN];
  int ncol[C::TN];
#pragma unroll
  for (int j = 0; j < C::TN; ++j) {
    int n = n0 + wn * C::WTN + j * 32 + r32;
    ncol[j] = n;
    bn[j] = n < N ? bf2f(bias[n]) : 0.f;
  }
  // EPI_QKV: per-column destination (which tensor, head, d)
  int qs[C::TN], qh[C::TN], qd[C::TN];
  if (EPI == EPI_QKV) {
#pragma unroll
    for (int j = 0; j < C::TN; ++j) {
      int n = ncol[j];
      int s = n / P.hidden, rem = n - s * P.hidden;
      qs[j] = s;
      qh[j] = rem / P.head_dim;
      qd[j] = rem - qh[j] * P.head_dim;
    }
  }
  const int rpb = P.rows_per_batch;
#pragma unroll
  for (int i = 0; i < C::TM; ++i) {
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) {
        const int m = m0 + wm * C::WTM + i * 32 + jj * 8 + g * 4 + ii;
        if (m >= M) continue;
        const int b = m / rpb;
        const int e = jj * 4 + ii;
        if (EPI == EPI_RESID) {
          float* __restrict__ xr = P.resid + (long)m * N;
          const float* __restrict__ gr = P.gate + (long)b * P.gate_stride;
#pragma unroll
          for (int j = 0; j < C::TN; ++j) {
            int n = ncol[j];
            if (n < N) xr[n] = xr[n] + gr[n] * (acc[i][j][e] + bn[j]);
          }
        } else if (EPI == EPI_GELU) {
          bf16_t* __restrict__ orow = (bf16_t*)P.out + (long)m * N;
#pragma unroll
          for (int j = 0; j < C::TN; ++j) {
            int n = ncol[j];
            if (n < N) orow[n] = f2bf(gelu_tanh(acc[i][j][e] + bn[j]));
          }
        } else if (EPI == EPI_STORE) {
          float* __restrict__ orow = (float*)P.out + (long)m * N;
#pragma unroll
          for (int j = 0; j < C::TN; ++j) {
            int n = ncol[j];
            if (n < N) orow[n] = acc[i][j][e] + bn[j];
          }
        } else {  // EPI_QKV
          const int jpos = m - b * rpb + P.seq_off;
#pragma unroll
          for (int j = 0; j < C::TN; ++j) {
            int n = ncol[j];
            if (n >= N) continue;
            bf16_t val = f2bf(acc[i][j][e] + bn[j]);
            long bh = (long)b * P.heads + qh[j];
            if (qs[j] == 0)
              ((bf16_t*)P.q)[(bh * P.Tj + jpos) * P.head_dim + qd[j]] = val;
            else if (qs[j] == 1)
              ((bf16_t*)P.k)[(bh * P.Tj + jpos) * P.head_dim + qd[j]] = val;
            else
              ((bf16_t*)P.v)[(bh * P.head_dim + qd[j]) * P.Tj_pad + jpos] = val;
          }
        }
      }
    }
  }
}

void gemm_tile_dims(int tile_cfg, int* bm, int* bn) {
  switch (tile_cfg) {
    case TILE_64x128: *bm = 64; *bn = 128; break;
    case TILE_128x64: *bm = 128; *bn = 64; break;
    case TILE_64x64: *bm = 64; *bn = 64; break;
    default: *bm = 128; *bn = 128; break;
  }
}

template <int BM, int BN>
static hipError_t launch_tile(const GemmArgs& a, int epi, hipStream_t st) {
  dim3 grid(a.total_tiles), block(256);
  switch (epi) {
    case EPI_QKV: hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, EPI_QKV>), grid, block, 0, st, a); break;
    case EPI_GELU: hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, EPI_GELU>), grid, block, 0, st, a); break;
    case EPI_RESID: hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, EPI_RESID>), grid, block, 0, st, a); break;
    default: hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, EPI_STORE>), grid, block, 0, st, a); break;
  }
  return hipGetLastError();
}

hipError_t launch_gemm_bf16(const GemmArgs& a, int epi, int tile_cfg, hipStream_t st) {
  switch (tile_cfg) {
    case TILE_64x128: return launch_tile<64, 128>(a, epi, st);
    case TILE_128x64: return launch_tile<128, 64>(a, epi, st);
    case TILE_64x64: return launch_tile<64, 64>(a, epi, st);
    default: return launch_tile<128, 128>(a, epi, st);
  }
}

}  // namespace ditmi
