// Internal launch interface between the host sequencer (ditmi.cpp) and the
// gfx950 kernels.  Argument structs are passed to kernels by value.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ditmi {

// ------------------------------------------------------------------ GEMM
// y[M, N] = A[M, K] * W[N, K]^T (+ bias), K-contiguous operands, then one of:
enum Epi {
  EPI_QKV = 0,    // +bias; scatter into head-major q, k and (bf16: transposed) v
  EPI_GELU = 1,   // +bias; tanh-GELU; store in the operand type
  EPI_RESID = 2,  // +bias; resid[m, n] += gate[b, n] * y   (fp32 residual stream)
  EPI_STORE = 3,  // +bias; store fp32
  EPI_RESID2 = 4  // as EPI_RESID; a separate instantiation so the MLP's second
                  // GEMM is a distinct kernel symbol in profiles
};

struct GemmProb {
  const void* A;      // [M, K]
  const void* W;      // [N, K]
  const void* bias;   // [N]
  int M, N, K;
  int tiles_m, tiles_n, tile_begin;
  int group_m;         // tile order: groups of group_m M-tiles x all N-tiles, M fastest (>= 1)
  int rows_per_batch;  // sample index b = m / rows_per_batch
  // EPI_RESID
  float* resid;
  const float* gate;   // gate[b * gate_stride + n]
  int gate_stride;
  // EPI_GELU / EPI_STORE
  void* out;           // [M, N] row-major
  // EPI_QKV: row m -> (b, j = m % rows_per_batch + seq_off) of the joint sequence
  void* q;             // [B, H, Tj, qk_stride]
  void* k;             // [B, H, Tj, qk_stride]
  void* v;             // bf16: v^T [B, H, dh, Tj_pad], key j at column v_key_pos(j); fp32: [B, H, Tj, dh]
  int seq_off, Tj, Tj_pad, heads, head_dim, hidden;
  int qk_stride;       // q/k row length: head_dim, or (bf16) head_dim rounded up to 16, padded with
                       // zeros except k's column head_dim, which holds 1
  float k_scale;       // bf16: k is stored multiplied by this (log2(e)/sqrt(dh), the softmax's exp2 scale)
  // Split K (bf16; EPI_GELU, EPI_RESID, EPI_RESID2): ksplit > 1 divides the
  // k-slices into ksplit equal ranges; the unit of tile t and range s stores
  // its fp32 product without bias to part[s][M][N], and
  // launch_splitk_gelu_bf16 / launch_splitk_resid then add the ranges and
  // apply the epilogue.
  float* part;
  int ksplit;
};

struct GemmArgs {
  GemmProb p[2];
  int nprob;
  int total_tiles;
  // Tail schedule (set with p[1].ksplit > 1): the tile counts of both
  // problems are multiples of 8, and every XCD runs its share of problem 0's
  // tiles before its share of problem 1's units, so the short split units
  // fill the last round instead of whole tiles.
  int tail;
};

// Column of key j in a bf16 v^T row: within each group of 16 keys the
// order is [0..3, 8..11, 4..7, 12..15] (bits 2 and 3 of j swapped), so the
// eight keys one lane of the attention PV MFMA needs (16c + 4g + 0..3 and
// 16c + 8 + 4g + 0..3) are one contiguous 16-byte chunk.  Tj_pad is a
// multiple of 16.
__host__ __device__ __forceinline__ int v_key_pos(int j) { return (j & ~12) | ((j & 4) << 1) | ((j & 8) >> 1); }

// ------------------------------------------------------------------ attention
struct AttnArgs {
  const void* q;   // bf16: [B, H, Tj, round16(dh)] zero padded; fp32: [B, H, Tj, dh]
  const void* k;   // same layout as q; bf16 with padding: column dh holds 1
  const void* v;   // bf16: v^T [B, H, dh, Tj_pad] (key j at column v_key_pos(j)); fp32: [B, H, Tj, dh]
  void* o;         // stream-major rows: image b*T + t, then text B*T + b*Tt + t; [*, H*dh]
  int B, H, Tj, Tj_pad, T_img, T_txt, D;
  float scale_log2;  // factor from q.k to the exp2 domain: log2(e) / sqrt(dh), or 1 where k is stored pre-scaled (bf16)
  float scale;       // 1 / sqrt(dh)
  // bf16 pipelined kernel, last partial round (attn_split_plan): the first
  // n_full (query block, head, sample) items run over all keys; each of the
  // n_tail items after them runs as `split` units over consecutive ranges of
  // key tiles, which store unnormalised partial results to `part`, and a
  // merge pass combines them.  split = 1: every item runs whole.
  int n_full, n_tail, split;
  float* part;  // [split][n_tail][256 queries][dh + 4] fp32: O (relative to the unit's m), m, l
};

// Plan of the pipelined attention's last round for B samples, H heads, Tj
// tokens: n_full items whole, n_tail items split into `split` key ranges.
// Returns the bytes of partial results it needs (0 without a split); a plan
// whose partials would exceed part_cap bytes is not used.
size_t attn_split_plan(int B, int H, int Tj, int head_dim, size_t part_cap, int* n_full, int* n_tail, int* split);

// ------------------------------------------------------------------ LayerNorm + modulate
struct LnSeg {
  const float* x;       // [rows, D] fp32
  void* out;            // [rows, D] operand type
  const float* shift;   // shift[b * mod_stride + n]
  const float* scale;   // scale[b * mod_stride + n]
  int rows, rows_per_batch, mod_stride, row_begin;
};
struct LnArgs {
  LnSeg s[2];
  int nseg, D, total_rows;
  float eps;
};

// ------------------------------------------------------------------ adaLN GEMV
constexpr int ADA_MAX_ENTRIES = 64;
constexpr int ADA_ROWS_PER_WG = 256;  // bf16 MFMA kernel: output rows per workgroup (the fp32 kernel: 128)
struct AdaEntry {
  const void* W;     // [N, D]
  const void* bias;  // [N]
  float* out;        // [B, N]
  int N, wg_begin;
};
struct AdaArgs {
  AdaEntry e[ADA_MAX_ENTRIES];
  int ne, total_wg;
  const float* cond;  // [B, D]
  const void* act;    // bf16 path: SiLU(cond) as bf16 [round16(B), D], zero rows past B
  int B, D;
};

// ------------------------------------------------------------------ launchers
// Each returns hipSuccess or the launch error.  dtype: 0 = fp32, 1 = bf16.
hipError_t launch_gemm_bf16(const GemmArgs& a, int epi, int tile_cfg, hipStream_t st);
// out[m][n] = bf16(GELU(sum_{s < S} part[s][m][n] + bias[n])), ranges added in
// order s = 0, 1, ...; M * N elements, N a multiple of 4.
hipError_t launch_splitk_gelu_bf16(const float* part, int S, int M, int N, const void* bias, void* out,
                                   hipStream_t st);
// resid[m][n] += gate[b * gate_stride + n] * (sum_{s < S} part[s][m][n] + bias[n]),
// b = m / rows_per_batch, ranges added in order s = 0, 1, ...; bf16 bias.
hipError_t launch_splitk_resid(const float* part, int S, int M, int N, const void* bias, const float* gate,
                               int gate_stride, int rows_per_batch, float* resid, hipStream_t st);
hipError_t launch_gemm_f32(const GemmArgs& a, int epi, hipStream_t st);
hipError_t launch_attn_bf16(const AttnArgs& a, int head_dim, hipStream_t st);
hipError_t launch_attn_f32(const AttnArgs& a, int head_dim, hipStream_t st);
hipError_t launch_ln_mod(const LnArgs& a, int dtype, hipStream_t st);
hipError_t launch_adaln(const AdaArgs& a, int dtype, hipStream_t st);
// act[r][k] = bf16(SiLU(cond[r][k])) for r < B, 0 for B <= r < round16(B)
hipError_t launch_silu_bf16(int B, int D, const float* cond, void* act, hipStream_t st);
hipError_t launch_cond_embed(int B, int D, const float* t, const int32_t* y, const void* w1, const void* b1,
                             const void* w2, const void* b2, const void* table, float* feat, float* h1,
                             float* cond, int dtype, hipStream_t st);
hipError_t launch_patch_embed(int rows, int T, int P, int D, const float* z, const void* w, const void* b,
                              const float* pos, float* x, int dtype, hipStream_t st);
hipError_t launch_pos_embed_2d(int gh, int gw, int D, float* pos, hipStream_t st);
hipError_t launch_fill_f32(float* p, int n, float v, hipStream_t st);
// z[i] += a * v[i], i < n; n a multiple of 4, both 16-byte aligned
hipError_t launch_axpy_f32(float* z, const float* v, float a, long n, hipStream_t st);

// Tile configurations of the bf16 GEMM (BM x BN, LDS ring depth).
enum {
  TILE_128x128 = 0, TILE_64x128 = 1, TILE_64x128_S2 = 2, TILE_64x144 = 3,
  TILE_256x256 = 4, TILE_256x128 = 5, TILE_256x192 = 6,
  TILE_64x144_1 = 7,  // 64 x 144 with one k-group of six waves (two workgroups per CU)
  TILE_COUNT = 8
};
void gemm_tile_dims(int tile_cfg, int* bm, int* bn);

}  // namespace ditmi
