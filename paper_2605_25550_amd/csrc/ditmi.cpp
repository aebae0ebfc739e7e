// Host side of the DiT-step library: C ABI, argument validation, workspace
// layout, GEMM tile planning and the launch sequence of a block and a step.
// Every argument is checked before the first launch, so a failing call
// enqueues nothing.  The library allocates no device memory: all tensors and
// the workspace belong to the caller.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <chrono>
#include <mutex>
#include <thread>
#include <string>
#include <vector>

#include "ditmi.h"
#include "kernels.h"

using namespace ditmi;

namespace {

thread_local std::string g_err;

dit_status fail(dit_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
inline bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }
inline long rup(long x, long m) { return (x + m - 1) / m * m; }

// ------------------------------------------------------------------ validation
dit_status check_shape(const dit_shape* s, bool step) {
  if (!s) return fail(DIT_ERR_INVALID_ARG, "shape is NULL");
  if (s->batch < 1 || s->tokens < 1 || s->text_tokens < 0)
    return fail(DIT_ERR_INVALID_ARG, "batch (%d) and tokens (%d) must be >= 1, text_tokens (%d) >= 0", s->batch,
                s->tokens, s->text_tokens);
  if (s->hidden < 64 || s->hidden % 64 != 0)
    return fail(DIT_ERR_INVALID_ARG, "hidden (%d) must be a positive multiple of 64", s->hidden);
  if (s->hidden > 4096) return fail(DIT_ERR_UNSUPPORTED, "hidden %d > 4096 is not supported", s->hidden);
  if (s->heads < 1 || s->head_dim < 1) return fail(DIT_ERR_INVALID_ARG, "heads and head_dim must be >= 1");
  if ((long)s->heads * s->head_dim != s->hidden)
    return fail(DIT_ERR_INVALID_ARG, "heads*head_dim (%d*%d) != hidden (%d)", s->heads, s->head_dim, s->hidden);
  if (s->head_dim != 64 && s->head_dim != 72 && s->head_dim != 128)
    return fail(DIT_ERR_UNSUPPORTED, "head_dim %d not supported (64, 72, 128)", s->head_dim);
  if (s->mlp_hidden < 64 || s->mlp_hidden % 64 != 0)
    return fail(DIT_ERR_INVALID_ARG, "mlp_hidden (%d) must be a positive multiple of 64", s->mlp_hidden);
  if (s->dtype != DIT_F32 && s->dtype != DIT_BF16) return fail(DIT_ERR_INVALID_ARG, "dtype %d unknown", s->dtype);
  if (!(s->ln_eps > 0.f) || !isfinite(s->ln_eps)) return fail(DIT_ERR_INVALID_ARG, "ln_eps must be finite and > 0");
  const long rows = (long)s->batch * (s->tokens + s->text_tokens);
  const long widest = s->mlp_hidden > 3 * s->hidden ? s->mlp_hidden : 3L * s->hidden;
  if (rows * widest >= (1L << 31) || rows >= (1L << 24))
    return fail(DIT_ERR_UNSUPPORTED, "batch*tokens (%ld rows) too large", rows);
  // The GEMM's DMA lane offsets (row * K * 2 bytes) and the adaLN/GEMV row
  // offsets are 32-bit: every weight matrix stays below 2^31 elements.  The
  // largest are fc1 / fc2 with F * D elements (w_ada 6 D^2 and w_qkv 3 D^2
  // are bounded by hidden <= 4096).
  if ((long)s->mlp_hidden * s->hidden >= (1L << 31))
    return fail(DIT_ERR_UNSUPPORTED, "mlp_hidden * hidden (%d * %d) >= 2^31 elements: weight matrix too large",
                s->mlp_hidden, s->hidden);
  if (step) {
    if (s->n_blocks < 1) return fail(DIT_ERR_INVALID_ARG, "n_blocks (%d) must be >= 1", s->n_blocks);
    if (s->patch_in < 1 || s->patch_in > 256 || s->patch_out < 4 || s->patch_out > 256 || s->patch_out % 4 != 0)
      return fail(DIT_ERR_INVALID_ARG, "patch_in (%d) must be in [1, 256] and patch_out (%d) a multiple of 4 in [4, 256]",
                  s->patch_in, s->patch_out);
  }
  return DIT_OK;
}

struct Layout {
  size_t mod, act, h, q, k, v, o, g, x, feat, h1, total;
  size_t t, vel, cond, xt;  // sampler loop: timesteps [B], velocity [B,T,P], c [B,D], text states [B,Tt,D]
  size_t slot_z[2], slot_y[2], slot_c[2];  // serving: two request slots
  size_t qk;  // q/k row length (elements)
  size_t part, part_cap;  // fp32 partials of split GEMMs: the dead q/k/v region, or a region of its own
  int ns, Tj, Tj_pad;
};

int choose_tile(const GemmProb* p, int np, int epi, size_t part_cap, int* split);

// Bytes of fp32 partials the split GEMMs of this shape need (the largest of
// the output projection, fc1 and fc2; 0 if none is split).
static size_t split_part_bytes(const dit_shape* s) {
  if (s->dtype != DIT_BF16) return 0;
  const int ns = s->text_tokens > 0 ? 2 : 1;
  const int D = s->hidden, F = s->mlp_hidden;
  const int gemms[3][3] = {{EPI_RESID, D, D}, {EPI_GELU, F, D}, {EPI_RESID2, D, F}};  // epilogue, N, K
  size_t need = 0;
  for (const auto& g : gemms) {
    GemmProb p[2] = {};
    for (int i = 0; i < ns; ++i) {
      p[i].M = s->batch * (i ? s->text_tokens : s->tokens);
      p[i].N = g[1];
      p[i].K = g[2];
      p[i].hidden = D;
    }
    int S = 0;
    choose_tile(p, ns, g[0], SIZE_MAX, &S);
    const size_t b = (size_t)S * p[ns - 1].M * p[ns - 1].N * 4;
    if (b > need) need = b;
  }
  return need;
}

Layout layout(const dit_shape* s, int kind) {
  Layout L{};
  const size_t E = s->dtype == DIT_BF16 ? 2 : 4;
  const size_t B = s->batch, T = s->tokens, Tt = s->text_tokens, D = s->hidden, F = s->mlp_hidden;
  const size_t H = s->heads, dh = s->head_dim;
  L.ns = Tt > 0 ? 2 : 1;
  L.Tj = (int)(T + Tt);
  L.Tj_pad = (int)rup(L.Tj, 16);  // v^T rows: whole 16-key groups (kernels.h: v_key_pos)
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off += align256(bytes);
    return o;
  };
  if (kind == DIT_WS_COND) {
    L.feat = take(B * 256 * 4);
    L.h1 = take(B * D * 4);
    L.total = off;
    return L;
  }
  const size_t rows = B * (T + Tt);
  const bool step = kind == DIT_WS_STEP || kind == DIT_WS_SAMPLE || kind == DIT_WS_SERVE;
  const size_t nmod = step ? (size_t)s->n_blocks * L.ns * B * 6 * D + B * 2 * D : L.ns * B * 6 * D;
  L.mod = take(nmod * 4);
  L.act = take((B + 15) / 16 * 16 * D * 2);  // SiLU(c) in bf16 for the adaLN MFMA kernel
  L.h = take(rows * D * E);
  L.qk = E == 2 ? (dh + 15) / 16 * 16 : dh;  // bf16 q/k rows are zero padded to whole MFMA k-steps
  L.q = take(B * H * L.Tj * L.qk * E);
  L.k = take(B * H * L.Tj * L.qk * E);
  L.v = take(E == 2 ? B * H * dh * (size_t)L.Tj_pad * 2 : B * H * L.Tj * dh * 4);
  L.o = take(rows * D * E);
  L.g = take(rows * F * E);
  {
    const size_t need = split_part_bytes(s), span = L.o - L.q;
    L.part = need <= span ? L.q : take(need);
    L.part_cap = need <= span ? span : need;
  }
  L.x = step ? take(B * T * D * 4) : 0;
  if (kind == DIT_WS_SAMPLE || kind == DIT_WS_SERVE) {
    L.t = take(B * 4);
    L.vel = take(B * T * (size_t)s->patch_out * 4);
    L.cond = take(B * D * 4);
    L.feat = take(B * 256 * 4);
    L.h1 = take(B * D * 4);
    L.xt = take(B * Tt * D * 4);
  }
  if (kind == DIT_WS_SERVE)
    for (int k = 0; k < 2; ++k) {
      L.slot_z[k] = take(B * T * (size_t)s->patch_out * 4);
      L.slot_y[k] = take(B * 4);
      L.slot_c[k] = take(B * D * 4);
    }
  L.total = off;
  return L;
}

dit_status check_stream_weights(const dit_stream_weights& w, const char* which) {
  const void* mats[] = {w.w_ada, w.w_qkv, w.w_o, w.w_fc1, w.w_fc2};
  const void* vecs[] = {w.b_ada, w.b_qkv, w.b_o, w.b_fc1, w.b_fc2};
  for (const void* p : mats)
    if (!p || !aligned(p, 16)) return fail(DIT_ERR_INVALID_ARG, "%s weight matrix NULL or not 16-byte aligned", which);
  for (const void* p : vecs)
    if (!p || !aligned(p, 16)) return fail(DIT_ERR_INVALID_ARG, "%s bias NULL or not 16-byte aligned", which);
  return DIT_OK;
}

// ------------------------------------------------------------------ timing hook
struct Timing {
  std::mutex mu;
  int kclass = -1, max = 0, used = 0;
  std::vector<hipEvent_t> ev;
  double flops = 0, bytes = 0;
} g_timing;

template <typename Fn>
hipError_t timed(int kclass, double flops, double bytes, hipStream_t st, Fn&& launch) {
  bool rec = false;
  int slot = 0;
  {
    std::lock_guard<std::mutex> lk(g_timing.mu);
    if (g_timing.kclass == kclass && g_timing.used < g_timing.max) {
      rec = true;
      slot = g_timing.used++;
      g_timing.flops += flops;
      g_timing.bytes += bytes;
    }
  }
  if (rec) {
    hipError_t e = hipEventRecord(g_timing.ev[2 * slot], st);
    if (e != hipSuccess) return e;
  }
  hipError_t e = launch();
  if (e != hipSuccess) return e;
  if (rec) return hipEventRecord(g_timing.ev[2 * slot + 1], st);
  return hipSuccess;
}

// ------------------------------------------------------------------ GEMM planning
struct Gemm {
  GemmArgs a{};
  int epi = EPI_STORE;
  int kclass = DIT_K_OTHER;
  double flops = 0, bytes = 0;
  float* part = nullptr;  // fp32 scratch for a split problem, part_cap bytes
  size_t part_cap = 0;
};

// bf16 tile choice, from per-shape measurements on MI355X (256 CUs).
// Per CU, the 256-row tiles (eight waves, one workgroup per CU) are the most
// efficient: a CU fetches (BM + BN) / (BM BN) bytes per flop, 1/128 for
// 256 x 256 against 1/64 for 128 x 128, and its LDS reads per flop are lower
// too.  Among 256 x 256, 256 x 192 and 256 x 128 the estimate
//   rounds of 256 tiles x BM x BN / efficiency
// decides, with relative per-CU efficiencies 1, 0.97 and 0.87 measured on
// the DiT shapes (ties go to the larger tile).  256 x 192 is not used
// with the residual epilogue (it would spill registers), nor beyond two
// rounds (measured slower there, e.g. the joint DiT's fc1 at 4352 rows:
// 8.48 ms per step against 7.86 ms with 256 x 256).  N a multiple of
// 144 with 193..256 tiles of 64 x 144 (DiT-XL/2 at 256 tokens x 8: the
// output projection and fc2) gets one balanced round of those first.
// Problems with fewer than 128 tiles of 256 x 128 use the 128 x 128 /
// 64 x 128 rules: 128 x 128 (two workgroups per CU) for 256..511 and >= 768
// tiles of 128 x 128, 64 x 128 with a 2-slot ring (three per CU) for
// 512..767, and 64 x 128 with a 3-slot ring below 256.
// The QKV epilogue needs tiles that do not straddle the k | v boundary at
// column 2D, i.e. BN dividing 2D.
static double tile_rounds(long tiles) { return (double)((tiles + 255) / 256); }

// Tail schedule: where problem 0 fills whole rounds of 256 tiles and the few
// tiles of problem 1 would take a round of their own (the joint block's fc1:
// 768 image + 48 text tiles of 256 x 256), problem 1 is split into S equal
// k-ranges (each at least 4 slices) whose S-times-shorter units fill that
// round, and a reduction adds the ranges.  Returns S, or 0 for no split.
static int tail_split(const GemmProb* p, int np, int epi, int bm, int bn, size_t part_cap) {
  if (np != 2 || (epi != EPI_GELU && epi != EPI_RESID && epi != EPI_RESID2) || part_cap == 0) return 0;
  const long t0 = (long)((p[0].M + bm - 1) / bm) * ((p[0].N + bn - 1) / bn);
  const long t1 = (long)((p[1].M + bm - 1) / bm) * ((p[1].N + bn - 1) / bn);
  if (t0 < 256 || t0 % 256 != 0 || t1 == 0 || 2 * t1 > 256) return 0;
  const int ks = p[1].K / 64;
  for (int S = 8; S >= 2; --S)
    if (t1 * S <= 256 && ks % S == 0 && ks / S >= 4 && (t1 * S) % 8 == 0 &&
        (size_t)S * p[1].M * p[1].N * 4 <= part_cap)
      return S;
  return 0;
}

// Cost of the split tail in rounds: the short units plus their fixed costs
// (prologue, fp32 partial stores, the reduction launch), estimated at 0.15
// of a round.
static double tail_rounds(long t0, int S) { return (double)(t0 / 256) + 1.0 / S + 0.15; }

// Fill split: a single problem whose tiles cannot fill the GPU is split
// into S equal k-ranges of at least 4 slices, e.g. the DiT-XL/2 fc2 at one
// sample of 256 tokens: 36 tiles of 64 x 128, each 72 k-slices long, as 216
// units of 12 slices.  Up to 128 tiles the units are at most one per CU
// (256; measured faster than more, smaller units sharing CUs); up to half
// of `slots` (the workgroups resident at once: 256 CUs x workgroups per CU)
// they may fill the slots.  S is the largest such split for which the
// estimated gain
//   (1 - 1/S) * 0.45 us per slice - partial traffic at 5 TB/s - 3 us
// of reduction launch is positive.  Returns S (0: no split).
static int fill_split(const GemmProb& p, int epi, int bm, int bn, long slots, size_t part_cap) {
  if ((epi != EPI_GELU && epi != EPI_RESID && epi != EPI_RESID2) || part_cap == 0) return 0;
  const long t = (long)((p.M + bm - 1) / bm) * ((p.N + bn - 1) / bn);
  const int ks = p.K / 64;
  if (t == 0 || 2 * t > slots) return 0;
  const long units = t <= 128 ? 256 : slots;
  for (int S = 8; S >= 2; --S) {
    if (t * S > units || ks % S != 0 || ks / S < 4 || (size_t)S * p.M * p.N * 4 > part_cap) continue;
    const double mn = (double)p.M * p.N;
    const double gain_us = (1.0 - 1.0 / S) * ks * 0.45 - (S * 4.0 + 8.0) * mn / 5e6 - 3.0;
    if (gain_us > 0) return S;
  }
  return 0;
}

int choose_tile(const GemmProb* p, int np, int epi, size_t part_cap, int* split) {
  *split = 0;
  long t128 = 0, t144 = 0, t256 = 0, t2x1 = 0, t192 = 0;
  bool n144 = true, ok256 = true, ok128 = true, ok192 = epi != EPI_RESID && epi != EPI_RESID2;
  for (int i = 0; i < np; ++i) {
    const long M = p[i].M, N = p[i].N;
    t128 += ((M + 127) / 128) * ((N + 127) / 128);
    t144 += ((M + 63) / 64) * (N / 144);
    t256 += ((M + 255) / 256) * ((N + 255) / 256);
    t2x1 += ((M + 255) / 256) * ((N + 127) / 128);
    t192 += ((M + 255) / 256) * ((N + 191) / 192);
    n144 = n144 && N % 144 == 0 && (epi != EPI_QKV || (2 * p[i].hidden) % 144 == 0);
    ok256 = ok256 && (epi != EPI_QKV || (2 * p[i].hidden) % 256 == 0);
    ok192 = ok192 && (epi != EPI_QKV || (2 * p[i].hidden) % 192 == 0);
    ok128 = ok128 && (epi != EPI_QKV || (2 * p[i].hidden) % 128 == 0);
  }
  if (n144 && t144 > 192 && t144 <= 256) return TILE_64x144;
  if (t2x1 >= 128) {
    int best = -1, best_split = 0;
    double best_cost = 0.0;
    auto consider = [&](bool ok, int cfg, long tiles, double area_over_eff) {
      int bm = 0, bn = 0;
      gemm_tile_dims(cfg, &bm, &bn);
      const int S = tail_split(p, np, epi, bm, bn, part_cap);
      const long t0 = (long)((p[0].M + bm - 1) / bm) * ((p[0].N + bn - 1) / bn);
      const double c = (S ? tail_rounds(t0, S) : tile_rounds(tiles)) * area_over_eff;
      if (ok && (best < 0 || c < best_cost)) best = cfg, best_cost = c, best_split = S;
    };
    consider(ok256, TILE_256x256, t256, 256.0 * 256.0 / 1.0);
    consider(ok192 && t192 <= 512, TILE_256x192, t192, 256.0 * 192.0 / 0.97);
    consider(ok128, TILE_256x128, t2x1, 256.0 * 128.0 / 0.87);
    if (best >= 0) {
      *split = best_split;
      return best;
    }
  }
  const int cfg = ((t128 >= 256 && t128 < 512) || t128 >= 768) ? TILE_128x128
                  : t128 >= 512                                   ? TILE_64x128_S2
                                                                  : TILE_64x128;
  if (np == 1) {
    int bm = 0, bn = 0;
    gemm_tile_dims(cfg, &bm, &bn);
    // resident workgroups per CU (LDS): 128x128 and 64x128 with 3 slots two, 64x128 with 2 slots three
    const long per_cu = cfg == TILE_64x128_S2 ? 3 : 2;
    *split = fill_split(p[0], epi, bm, bn, 256 * per_cu, part_cap);
  }
  return cfg;
}

// Row tail: a single problem of whole rounds of 256-row tiles plus a short
// last round (the video DiT's fc2 and output projection at 17550 tokens:
// 828 tiles of 256 x 256 = 3 rounds + 60 tiles) is cut after the last row
// tile that completes a round; the rows after it become the second problem
// of the tail schedule, whose tiles run as k-range units in the last round.
// Applies where the sample index of a row stays valid in the second part
// (one sample, or a cut at a sample boundary).  Returns the split (0: none;
// the problem is then unchanged).
static int row_tail(GemmArgs& a, int epi, int bm, int bn, size_t part_cap) {
  if (a.nprob != 1 || bm != 256 || (epi != EPI_GELU && epi != EPI_RESID && epi != EPI_RESID2)) return 0;
  const GemmProb& p = a.p[0];
  const long tm = (p.M + bm - 1) / bm, tn = (p.N + bn - 1) / bn;
  if (tm * tn <= 256 || (tm * tn) % 256 == 0) return 0;
  long m0 = 0;
  for (long m = tm - 1; m >= 1 && !m0; --m)
    if ((m * tn) % 256 == 0) m0 = m;
  if (!m0) return 0;
  const long M0 = m0 * bm, rpb = p.rows_per_batch;
  if (p.M > rpb && M0 % rpb != 0) return 0;
  GemmProb two[2] = {p, p};
  two[0].M = (int)M0;
  two[1].M = (int)(p.M - M0);
  const int S = tail_split(two, 2, epi, bm, bn, part_cap);
  if (!S || tail_rounds(m0 * tn, S) >= tile_rounds(tm * tn)) return 0;
  GemmProb& q = two[1];
  q.A = (const uint16_t*)p.A + M0 * p.K;  // bf16 elements
  q.rows_per_batch = (int)rpb;
  if (epi == EPI_GELU) {
    q.out = (uint16_t*)p.out + M0 * p.N;
  } else {
    q.resid = p.resid + M0 * p.N;
    q.gate = p.gate + (M0 / rpb) * p.gate_stride;
  }
  a.p[0] = two[0];
  a.p[1] = q;
  a.nprob = 2;
  return S;
}

// Height (in M-tiles) of the tile groups of the GEMM's tile order.  An XCD
// runs a contiguous range of that order, c tiles at a time (one per
// workgroup slot of its 32 CUs, or its whole share of a smaller grid); such
// a range spans about g M-tiles and c / g N-tiles, so it reads
// g BM rows of A and (c / g) BN rows of W per k-slice from the XCD's L2.
// The height with the least of that (ties: the taller) is used.  DiT-XL/2's
// QKV projection at 256 tokens x 8 (8 x 27 tiles of 256 x 128, 27 per XCD):
// 4 M-tiles x 7 N-tiles per XCD instead of 8 x 3.4.
// Where A is larger than the Infinity Cache can keep (its 256 MB hold W and
// what else the step touches; taken as 192 MB) and larger than W, every
// extra pass over A comes from HBM, while W stays cached: the height is then
// the one that lets an XCD's concurrent tiles span all N-tiles, so A is
// streamed once.  Video DiT fc2 (17550 x 12288 A, 431 MB): height 2, 1249 ->
// 1179 us per launch against the balanced 8.
static int group_height(int tiles_m, int tiles_n, int bm, int bn, int tcfg, double a_bytes, double w_bytes) {
  const long tiles = (long)tiles_m * tiles_n;
  const int per_cu = tcfg == TILE_128x128 || tcfg == TILE_64x128 || tcfg == TILE_64x144_1 ? 2
                     : tcfg == TILE_64x128_S2                                             ? 3
                                                                                          : 1;
  const long c = std::min<long>(32L * per_cu, (tiles + 7) / 8);
  if (a_bytes > 192e6 && a_bytes > w_bytes) return (int)std::max<long>(1, std::min<long>(tiles_m, c / tiles_n));
  int best = 8;
  double best_cost = -1;
  for (int g = 16; g >= 1; g /= 2) {
    const int gm = std::min(g, tiles_m);
    const double cost = (double)gm * bm + (double)((c + gm - 1) / gm) * bn;
    if (best_cost < 0 || cost < best_cost) best = gm, best_cost = cost;
  }
  return best < 1 ? 1 : best;
}

hipError_t run_gemm(Gemm& G, int dtype, hipStream_t st) {
  GemmArgs& a = G.a;
  int bm = 64, bn = 64, tcfg = 0, split = 0;
  if (dtype == DIT_BF16) {
    tcfg = choose_tile(a.p, a.nprob, G.epi, G.part_cap, &split);
    gemm_tile_dims(tcfg, &bm, &bn);
    if (!split) split = row_tail(a, G.epi, bm, bn, G.part_cap);
  }
  int tiles = 0;
  for (int i = 0; i < a.nprob; ++i) {
    GemmProb& p = a.p[i];
    p.tiles_m = (p.M + bm - 1) / bm;
    p.tiles_n = (p.N + bn - 1) / bn;
    const double esz = dtype == DIT_BF16 ? 2.0 : 4.0;
    p.group_m = group_height(p.tiles_m, p.tiles_n, bm, bn, dtype == DIT_BF16 ? tcfg : -1, esz * p.M * p.K,
                             esz * p.N * p.K);
    p.tile_begin = tiles;
    p.ksplit = 0;
    p.part = nullptr;
    tiles += p.tiles_m * p.tiles_n * (i == 1 && split ? split : 1);
  }
  // The split problem is the second of two (tail schedule) or the only one
  // (fill split, every unit in one round, the usual tile order).
  const int sp = a.nprob - 1;
  if (split && sp == 0) tiles *= split;
  a.total_tiles = tiles;
  a.tail = split && sp == 1 ? 1 : 0;
  if (split) {
    a.p[sp].ksplit = split;
    a.p[sp].part = G.part;
  }
  if (tiles == 0) return hipSuccess;
  hipError_t e = timed(G.kclass, G.flops, G.bytes, st, [&]() {
    return dtype == DIT_BF16 ? launch_gemm_bf16(a, G.epi, tcfg, st) : launch_gemm_f32(a, G.epi, st);
  });
  if (e != hipSuccess || !split) return e;
  const GemmProb& q = a.p[sp];
  const double mn = (double)q.M * q.N;
  if (G.epi == EPI_GELU)
    return timed(DIT_K_OTHER, 0, mn * (split * 4.0 + 2.0) + q.N * 2.0, st, [&]() {
      return launch_splitk_gelu_bf16(q.part, split, q.M, q.N, q.bias, q.out, st);
    });
  return timed(DIT_K_OTHER, 0, mn * (split * 4.0 + 8.0) + q.N * 2.0, st, [&]() {
    return launch_splitk_resid(q.part, split, q.M, q.N, q.bias, q.gate, q.gate_stride, q.rows_per_batch, q.resid, st);
  });
}

// ------------------------------------------------------------------ block sequence
struct StreamIO {
  const dit_stream_weights* w;
  float* x;           // residual [B, Ts, D]
  const float* mod;   // [B, 6D]
  int Ts;             // tokens of this stream per sample
};

#define HIP_TRY(expr)                                                                     \
  do {                                                                                    \
    hipError_t _e = (expr);                                                               \
    if (_e != hipSuccess) return fail(DIT_ERR_HIP, "%s: %s", #expr, hipGetErrorString(_e)); \
  } while (0)

dit_status run_block(const dit_shape* s, const Layout& L, char* ws, StreamIO* io, int ns, hipStream_t st) {
  const int B = s->batch, D = s->hidden, F = s->mlp_hidden, H = s->heads, dh = s->head_dim;
  const int dt = s->dtype;
  const size_t E = dt == DIT_BF16 ? 2 : 4;
  char* h = ws + L.h;
  char* o = ws + L.o;
  char* gbuf = ws + L.g;
  const long rows0 = (long)B * io[0].Ts;
  // row offsets of stream 1 inside the stream-major activation buffers
  auto act = [&](char* base, int si, long width) { return (void*)(base + (si ? rows0 * width * E : 0)); };

  auto ln = [&](int which) -> hipError_t {  // which 0: (shift1, scale1), 1: (shift2, scale2)
    LnArgs a{};
    a.nseg = ns;
    a.D = D;
    a.eps = s->ln_eps;
    long begin = 0;
    for (int i = 0; i < ns; ++i) {
      LnSeg& g = a.s[i];
      g.x = io[i].x;
      g.out = act(h, i, D);
      g.shift = io[i].mod + (which ? 3 : 0) * D;
      g.scale = io[i].mod + (which ? 4 : 1) * D;
      g.rows = B * io[i].Ts;
      g.rows_per_batch = io[i].Ts;
      g.mod_stride = 6 * D;
      g.row_begin = (int)begin;
      begin += g.rows;
    }
    a.total_rows = (int)begin;
    const double bytes = (double)begin * D * (4 + E);
    return timed(DIT_K_LN_MOD, 0, bytes, st, [&]() { return launch_ln_mod(a, dt, st); });
  };
  auto prob_common = [&](GemmProb& p, int i, const void* A, const void* W, const void* bias, int N, int K) {
    p.A = A;
    p.W = W;
    p.bias = bias;
    p.M = B * io[i].Ts;
    p.N = N;
    p.K = K;
    p.rows_per_batch = io[i].Ts;
  };
  double tokens = 0;
  for (int i = 0; i < ns; ++i) tokens += (double)B * io[i].Ts;

  // (1) h = LN(x) * (1 + scale1) + shift1
  HIP_TRY(ln(0));
  // (2) q, k, v = h W_qkv^T + b_qkv, scattered head-major
  {
    Gemm G;
    G.epi = EPI_QKV;
    G.kclass = DIT_K_GEMM_QKV;
    G.a.nprob = ns;
    for (int i = 0; i < ns; ++i) {
      GemmProb& p = G.a.p[i];
      prob_common(p, i, act(h, i, D), io[i].w->w_qkv, io[i].w->b_qkv, 3 * D, D);
      p.q = ws + L.q;
      p.k = ws + L.k;
      p.v = ws + L.v;
      p.seq_off = i ? io[0].Ts : 0;
      p.Tj = L.Tj;
      p.Tj_pad = L.Tj_pad;
      p.heads = H;
      p.head_dim = dh;
      p.hidden = D;
      p.qk_stride = (int)L.qk;
      p.k_scale = (float)(1.4426950408889634 / sqrt((double)dh));
    }
    G.flops = 2.0 * tokens * 3 * D * D;
    G.bytes = (tokens * D + ns * 3.0 * D * D + tokens * 3 * D) * E;
    HIP_TRY(run_gemm(G, dt, st));
  }
  // (3) o = softmax(q k^T / sqrt(dh)) v over the joint sequence
  {
    AttnArgs a{};
    a.q = ws + L.q;
    a.k = ws + L.k;
    a.v = ws + L.v;
    a.o = o;
    a.B = B;
    a.H = H;
    a.Tj = L.Tj;
    a.Tj_pad = L.Tj_pad;
    a.T_img = io[0].Ts;
    a.T_txt = ns > 1 ? io[1].Ts : 0;
    a.D = D;
    a.scale = 1.0f / sqrtf((float)dh);
    // the bf16 QKV epilogue stores k already in the exp2 domain
    a.scale_log2 = dt == DIT_BF16 ? 1.0f : (float)(1.4426950408889634 / sqrt((double)dh));
    // key-range split of the last partial round; its partial results use the
    // MLP hidden region g, which is dead until fc1
    if (dt == DIT_BF16) {
      const size_t g_bytes = (size_t)B * L.Tj * F * E;
      if (attn_split_plan(B, H, L.Tj, dh, g_bytes, &a.n_full, &a.n_tail, &a.split) > 0) a.part = (float*)gbuf;
    }
    const double flops = 4.0 * B * H * (double)L.Tj * L.Tj * dh;
    const double bytes = 4.0 * B * (double)L.Tj * D * E;
    HIP_TRY(timed(DIT_K_ATTENTION, flops, bytes, st, [&]() {
      return dt == DIT_BF16 ? launch_attn_bf16(a, dh, st) : launch_attn_f32(a, dh, st);
    }));
  }
  // (4) x += gate1 * (o W_o^T + b_o)
  {
    Gemm G;
    G.epi = EPI_RESID;
    G.kclass = DIT_K_GEMM_OUT;
    G.a.nprob = ns;
    for (int i = 0; i < ns; ++i) {
      GemmProb& p = G.a.p[i];
      prob_common(p, i, act(o, i, D), io[i].w->w_o, io[i].w->b_o, D, D);
      p.resid = io[i].x;
      p.gate = io[i].mod + 2 * D;
      p.gate_stride = 6 * D;
    }
    // fp32 partials of a split GEMM: q, k and v are dead after attention
    // (where their region is too small the workspace has one of its own)
    G.part = (float*)(ws + L.part);
    G.part_cap = L.part_cap;
    G.flops = 2.0 * tokens * D * D;
    G.bytes = (tokens * D + ns * (double)D * D) * E + tokens * D * 8.0;
    HIP_TRY(run_gemm(G, dt, st));
  }
  // (5) h = LN(x) * (1 + scale2) + shift2
  HIP_TRY(ln(1));
  // (6) g = GELU(h W_1^T + b_1)
  {
    Gemm G;
    G.epi = EPI_GELU;
    G.kclass = DIT_K_GEMM_FC1;
    G.a.nprob = ns;
    for (int i = 0; i < ns; ++i) {
      GemmProb& p = G.a.p[i];
      prob_common(p, i, act(h, i, D), io[i].w->w_fc1, io[i].w->b_fc1, F, D);
      p.out = act(gbuf, i, F);
    }
    G.part = (float*)(ws + L.part);
    G.part_cap = L.part_cap;
    G.flops = 2.0 * tokens * F * D;
    G.bytes = (tokens * D + ns * (double)F * D + tokens * F) * E;
    HIP_TRY(run_gemm(G, dt, st));
  }
  // (7) x += gate2 * (g W_2^T + b_2)
  {
    Gemm G;
    G.epi = EPI_RESID2;
    G.kclass = DIT_K_GEMM_FC2;
    G.a.nprob = ns;
    for (int i = 0; i < ns; ++i) {
      GemmProb& p = G.a.p[i];
      prob_common(p, i, act(gbuf, i, F), io[i].w->w_fc2, io[i].w->b_fc2, D, F);
      p.resid = io[i].x;
      p.gate = io[i].mod + 5 * D;
      p.gate_stride = 6 * D;
    }
    G.part = (float*)(ws + L.part);
    G.part_cap = L.part_cap;
    G.flops = 2.0 * tokens * D * F;
    G.bytes = (tokens * F + ns * (double)D * F) * E + tokens * D * 8.0;
    HIP_TRY(run_gemm(G, dt, st));
  }
  return DIT_OK;
}

// adaLN GEMVs for a list of (W, bias, out, N) in launches of <= 64 entries.
struct AdaJob {
  const void* W;
  const void* bias;
  float* out;
  int N;
};

dit_status run_adaln(const dit_shape* s, const float* cond, void* act, const std::vector<AdaJob>& jobs,
                     hipStream_t st) {
  const size_t E = s->dtype == DIT_BF16 ? 2 : 4;
  if (s->dtype == DIT_BF16)
    HIP_TRY(timed(DIT_K_OTHER, 0, 0, st, [&]() { return launch_silu_bf16(s->batch, s->hidden, cond, act, st); }));
  for (size_t j0 = 0; j0 < jobs.size(); j0 += ADA_MAX_ENTRIES) {
    AdaArgs a{};
    a.cond = cond;
    a.act = act;
    a.B = s->batch;
    a.D = s->hidden;
    int wg = 0;
    double bytes = 0;
    const size_t j1 = j0 + ADA_MAX_ENTRIES < jobs.size() ? j0 + ADA_MAX_ENTRIES : jobs.size();
    for (size_t j = j0; j < j1; ++j) {
      AdaEntry& e = a.e[a.ne++];
      e.W = jobs[j].W;
      e.bias = jobs[j].bias;
      e.out = jobs[j].out;
      e.N = jobs[j].N;
      e.wg_begin = wg;
      const int rows_per_wg = s->dtype == DIT_BF16 ? ADA_ROWS_PER_WG : 128;
      wg += (jobs[j].N + rows_per_wg - 1) / rows_per_wg;
      bytes += (double)jobs[j].N * s->hidden * E;
    }
    a.total_wg = wg;
    HIP_TRY(timed(DIT_K_ADALN, 2.0 * bytes / E * s->batch, bytes, st,
                  [&]() { return launch_adaln(a, s->dtype, st); }));
  }
  return DIT_OK;
}

// Validation shared by the step and the sampler loop: shape, step weights
// and every block's weights.
dit_status check_step_weights(const dit_shape* s, const dit_step_weights* w) {
  dit_status st = check_shape(s, true);
  if (st != DIT_OK) return st;
  if (!w || !w->blocks) return fail(DIT_ERR_INVALID_ARG, "step weights or block array is NULL");
  if (!w->w_patch || !w->b_patch || !w->w_ada_final || !w->b_ada_final || !w->w_final || !w->b_final)
    return fail(DIT_ERR_INVALID_ARG, "a step weight pointer is NULL");
  if (!aligned(w->w_ada_final, 16) || !aligned(w->w_final, 16) || !aligned(w->w_patch, 4) ||
      !aligned(w->b_final, 16))
    return fail(DIT_ERR_INVALID_ARG, "step weight misaligned (matrices and b_final need 16 bytes)");
  if (w->pos && !aligned(w->pos, 4)) return fail(DIT_ERR_INVALID_ARG, "pos misaligned");
  const bool joint = s->text_tokens > 0;
  for (int l = 0; l < s->n_blocks; ++l) {
    if ((st = check_stream_weights(w->blocks[l].img, "image-stream")) != DIT_OK) return st;
    if (joint && (st = check_stream_weights(w->blocks[l].txt, "text-stream")) != DIT_OK) return st;
  }
  return DIT_OK;
}

// One denoising step on validated arguments (the step part of the layout L
// of the workspace ws): adaLN for all blocks, patch embedding, blocks, final
// layer into out.
dit_status run_step(const dit_shape* s, const dit_step_weights* w, const Layout& L, char* ws, const float* patches,
                    float* x_txt, const float* cond, float* out, hipStream_t hs) {
  dit_status st = DIT_OK;
  const bool joint = s->text_tokens > 0;
  const int B = s->batch, T = s->tokens, D = s->hidden, ns = L.ns;
  float* mod = (float*)(ws + L.mod);
  const size_t per = (size_t)B * 6 * D;
  float* mod_final = mod + (size_t)s->n_blocks * ns * per;
  float* x = (float*)(ws + L.x);

  // (a2) every block's modulation vectors and the final layer's, hoisted
  std::vector<AdaJob> jobs;
  for (int l = 0; l < s->n_blocks; ++l) {
    jobs.push_back({w->blocks[l].img.w_ada, w->blocks[l].img.b_ada, mod + (size_t)(l * ns) * per, 6 * D});
    if (joint) jobs.push_back({w->blocks[l].txt.w_ada, w->blocks[l].txt.b_ada, mod + (size_t)(l * ns + 1) * per, 6 * D});
  }
  jobs.push_back({w->w_ada_final, w->b_ada_final, mod_final, 2 * D});
  if ((st = run_adaln(s, cond, ws + L.act, jobs, hs)) != DIT_OK) return st;

  // (a3) x = patches W_patch^T + b_patch (+ pos)
  HIP_TRY(timed(DIT_K_OTHER, 2.0 * B * T * D * s->patch_in, (double)B * T * (s->patch_in + D) * 4.0, hs, [&]() {
    return launch_patch_embed(B * T, T, s->patch_in, D, patches, w->w_patch, w->b_patch, w->pos, x, s->dtype, hs);
  }));

  // (a4-a11) blocks
  for (int l = 0; l < s->n_blocks; ++l) {
    StreamIO io[2] = {{&w->blocks[l].img, x, mod + (size_t)(l * ns) * per, T},
                      {&w->blocks[l].txt, x_txt, mod + (size_t)(l * ns + 1) * per, s->text_tokens}};
    if ((st = run_block(s, L, ws, io, ns, hs)) != DIT_OK) return st;
  }

  // (a12) out = (LN(x) * (1 + scale_f) + shift_f) W_final^T + b_final, image tokens only
  {
    LnArgs a{};
    a.nseg = 1;
    a.D = D;
    a.eps = s->ln_eps;
    a.total_rows = B * T;
    a.s[0] = LnSeg{x, ws + L.h, mod_final, mod_final + D, B * T, T, 2 * D, 0};
    HIP_TRY(timed(DIT_K_LN_MOD, 0, (double)B * T * D * 6.0, hs, [&]() { return launch_ln_mod(a, s->dtype, hs); }));
    Gemm G;
    G.epi = EPI_STORE;
    G.kclass = DIT_K_OTHER;
    G.a.nprob = 1;
    GemmProb& p = G.a.p[0];
    p.A = ws + L.h;
    p.W = w->w_final;
    p.bias = w->b_final;
    p.M = B * T;
    p.N = s->patch_out;
    p.K = D;
    p.rows_per_batch = T;
    p.out = out;
    G.flops = 2.0 * B * T * D * s->patch_out;
    HIP_TRY(run_gemm(G, s->dtype, hs));
  }
  return DIT_OK;
}

// The Euler loop of dit_sample_euler on validated arguments (sampler part of
// the layout L of ws): per step the conditioning (from cw and y at
// t_i = sigma_i * t_scale, or the given cond), the step into the velocity
// buffer, and z += (sigma_{i+1} - sigma_i) v.
dit_status run_sample_loop(const dit_shape* s, const dit_step_weights* w, const dit_cond_weights* cw,
                           const int32_t* y, const float* cond, const float* sigmas, int n_steps, float t_scale,
                           float* z, const float* x_txt, const Layout& L, char* ws, hipStream_t hs) {
  dit_status st = DIT_OK;
  const bool joint = s->text_tokens > 0;
  const int B = s->batch, D = s->hidden;
  const long nz = (long)B * s->tokens * s->patch_out;
  float* vel = (float*)(ws + L.vel);
  float* xt = joint ? (float*)(ws + L.xt) : nullptr;
  for (int i = 0; i < n_steps; ++i) {
    const float* c = cond;
    if (cw) {  // c_i = conditioning at t_i = sigma_i * t_scale (fp32), every sample
      const float t = sigmas[i] * t_scale;
      HIP_TRY(launch_fill_f32((float*)(ws + L.t), B, t, hs));
      HIP_TRY(timed(DIT_K_OTHER, 0, 0, hs, [&]() {
        return launch_cond_embed(B, D, (const float*)(ws + L.t), y, cw->w_t1, cw->b_t1, cw->w_t2, cw->b_t2,
                                 cw->class_table, (float*)(ws + L.feat), (float*)(ws + L.h1), (float*)(ws + L.cond),
                                 s->dtype, hs);
      }));
      c = (const float*)(ws + L.cond);
    }
    if (joint)  // every step starts from the given text states
      HIP_TRY(hipMemcpyAsync(xt, x_txt, (size_t)B * s->text_tokens * D * sizeof(float), hipMemcpyDeviceToDevice, hs));
    if ((st = run_step(s, w, L, ws, z, xt, c, vel, hs)) != DIT_OK) return st;
    const float dsig = sigmas[i + 1] - sigmas[i];
    HIP_TRY(timed(DIT_K_OTHER, 2.0 * nz, 12.0 * nz, hs, [&]() { return launch_axpy_f32(z, vel, dsig, nz, hs); }));
  }
  return DIT_OK;
}

// Arguments of a block call, everything but the workspace.
dit_status check_block_args(const dit_shape* s, const dit_block_weights* w, const float* x, const float* x_txt,
                            const float* cond) {
  dit_status st = check_shape(s, false);
  if (st != DIT_OK) return st;
  if (!w) return fail(DIT_ERR_INVALID_ARG, "weights is NULL");
  if ((st = check_stream_weights(w->img, "image-stream")) != DIT_OK) return st;
  const bool joint = s->text_tokens > 0;
  if (joint && (st = check_stream_weights(w->txt, "text-stream")) != DIT_OK) return st;
  if (!x || !aligned(x, 16)) return fail(DIT_ERR_INVALID_ARG, "x NULL or not 16-byte aligned");
  if (joint && (!x_txt || !aligned(x_txt, 16))) return fail(DIT_ERR_INVALID_ARG, "x_txt NULL or not 16-byte aligned");
  if (!joint && x_txt) return fail(DIT_ERR_INVALID_ARG, "x_txt must be NULL when text_tokens == 0");
  if (!cond || !aligned(cond, 4)) return fail(DIT_ERR_INVALID_ARG, "cond NULL or misaligned");
  return DIT_OK;
}

// One block on validated arguments: adaLN of the block's stream(s), then
// the block, with the block layout L of the workspace ws.
dit_status block_call(const dit_shape* s, const dit_block_weights* w, float* x, float* x_txt, const float* cond,
                      const Layout& L, char* ws, hipStream_t hs) {
  const bool joint = s->text_tokens > 0;
  float* mod = (float*)(ws + L.mod);
  const size_t per = (size_t)s->batch * 6 * s->hidden;
  std::vector<AdaJob> jobs;
  jobs.push_back({w->img.w_ada, w->img.b_ada, mod, 6 * s->hidden});
  if (joint) jobs.push_back({w->txt.w_ada, w->txt.b_ada, mod + per, 6 * s->hidden});
  dit_status st = run_adaln(s, cond, ws + L.act, jobs, hs);
  if (st != DIT_OK) return st;
  StreamIO io[2] = {{&w->img, x, mod, s->tokens}, {&w->txt, x_txt, mod + per, s->text_tokens}};
  return run_block(s, L, ws, io, joint ? 2 : 1, hs);
}

// ------------------------------------------------------------------ static scratch
// Workspace of dit_block_forward_noalloc: one array per GPU, in the code
// object's zero-initialised data, held until the process ends.  Host code
// never uses the array's name as an address (it stands for a host-side
// shadow); the device address comes from hipGetSymbolAddress, looked up
// once per device with that device current and kept in `scratch_ptr`.
// Every byte a block reads from its workspace is written first by the same
// call, so nothing is cleared between calls.
static __device__ __align__(256) unsigned char scratch[DIT_NOALLOC_SCRATCH_BYTES];

struct ScratchTable {
  std::mutex mu;
  std::vector<char*> ptr;  // per device ordinal; null until looked up
} g_scratch;

dit_status scratch_of_stream(hipStream_t hs, char** out) {
  int dev = -1;
  hipError_t e = hs ? hipStreamGetDevice(hs, &dev) : hipGetDevice(&dev);
  if (e != hipSuccess || dev < 0) return fail(DIT_ERR_HIP, "device of the stream: %s", hipGetErrorString(e));
  std::lock_guard<std::mutex> lk(g_scratch.mu);
  if ((int)g_scratch.ptr.size() <= dev) g_scratch.ptr.resize(dev + 1, nullptr);
  if (!g_scratch.ptr[dev]) {
    int cur = -1;
    HIP_TRY(hipGetDevice(&cur));
    if (cur != dev) HIP_TRY(hipSetDevice(dev));
    void* scratch_ptr = nullptr;
    e = hipGetSymbolAddress((void**)&scratch_ptr, HIP_SYMBOL(scratch));
    if (cur != dev) (void)hipSetDevice(cur);
    if (e != hipSuccess || !scratch_ptr)
      return fail(DIT_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
    g_scratch.ptr[dev] = (char*)scratch_ptr;
  }
  *out = g_scratch.ptr[dev];
  return DIT_OK;
}

}  // namespace

// ====================================================================== C ABI
extern "C" {

int dit_version(void) { return DITMI_VERSION; }

const char* dit_status_string(dit_status st) {
  switch (st) {
    case DIT_OK: return "ok";
    case DIT_ERR_INVALID_ARG: return "invalid argument";
    case DIT_ERR_UNSUPPORTED: return "unsupported shape";
    case DIT_ERR_WORKSPACE: return "workspace too small";
    case DIT_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

const char* dit_last_error(void) { return g_err.c_str(); }

size_t dit_workspace_bytes(const dit_shape* s, int kind) {
  if (kind < DIT_WS_BLOCK || kind > DIT_WS_SERVE) {
    fail(DIT_ERR_INVALID_ARG, "unknown workspace kind %d", kind);
    return 0;
  }
  if (check_shape(s, kind == DIT_WS_STEP || kind == DIT_WS_SAMPLE || kind == DIT_WS_SERVE) != DIT_OK) return 0;
  return layout(s, kind).total;
}

dit_status dit_block_forward(const dit_shape* s, const dit_block_weights* w, float* x, float* x_txt,
                             const float* cond, void* workspace, size_t ws_bytes, void* stream) {
  dit_status st = check_block_args(s, w, x, x_txt, cond);
  if (st != DIT_OK) return st;
  const Layout L = layout(s, DIT_WS_BLOCK);
  if (!workspace || !aligned(workspace, 256)) return fail(DIT_ERR_INVALID_ARG, "workspace NULL or not 256-byte aligned");
  if (ws_bytes < L.total) return fail(DIT_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", ws_bytes, L.total);
  return block_call(s, w, x, x_txt, cond, L, (char*)workspace, (hipStream_t)stream);
}

dit_status dit_block_forward_noalloc(const dit_shape* s, const dit_block_weights* w, float* x, float* x_txt,
                                     const float* cond, void* stream) {
  dit_status st = check_block_args(s, w, x, x_txt, cond);
  if (st != DIT_OK) return st;
  const Layout L = layout(s, DIT_WS_BLOCK);
  if (L.total > (size_t)DIT_NOALLOC_SCRATCH_BYTES)
    return fail(DIT_ERR_UNSUPPORTED,
                "dit_block_forward_noalloc: this block needs %zu bytes of scratch, above the %zu-byte static "
                "scratch; use dit_block_forward with a workspace",
                L.total, (size_t)DIT_NOALLOC_SCRATCH_BYTES);
  hipStream_t hs = (hipStream_t)stream;
  char* ws = nullptr;
  if ((st = scratch_of_stream(hs, &ws)) != DIT_OK) return st;
  return block_call(s, w, x, x_txt, cond, L, ws, hs);
}

dit_status dit_step_forward(const dit_shape* s, const dit_step_weights* w, const float* patches, float* x_txt,
                            const float* cond, float* out, void* workspace, size_t ws_bytes, void* stream) {
  dit_status st = check_step_weights(s, w);
  if (st != DIT_OK) return st;
  const bool joint = s->text_tokens > 0;
  if (!patches || !aligned(patches, 4)) return fail(DIT_ERR_INVALID_ARG, "patches NULL or misaligned");
  if (joint && (!x_txt || !aligned(x_txt, 16))) return fail(DIT_ERR_INVALID_ARG, "x_txt NULL or not 16-byte aligned");
  if (!joint && x_txt) return fail(DIT_ERR_INVALID_ARG, "x_txt must be NULL when text_tokens == 0");
  if (!cond || !aligned(cond, 4)) return fail(DIT_ERR_INVALID_ARG, "cond NULL or misaligned");
  if (!out || !aligned(out, 16)) return fail(DIT_ERR_INVALID_ARG, "out NULL or not 16-byte aligned");
  const Layout L = layout(s, DIT_WS_STEP);
  if (!workspace || !aligned(workspace, 256)) return fail(DIT_ERR_INVALID_ARG, "workspace NULL or not 256-byte aligned");
  if (ws_bytes < L.total) return fail(DIT_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", ws_bytes, L.total);
  return run_step(s, w, L, (char*)workspace, patches, x_txt, cond, out, (hipStream_t)stream);
}

dit_status dit_serve(const dit_shape* s, const dit_step_weights* w, const dit_cond_weights* cw,
                     const dit_request* reqs, int32_t n_requests, const float* sigmas, int32_t n_steps, float t_scale,
                     int32_t overlap, uint32_t jitter_us, uint32_t jitter_seed, void* workspace, size_t ws_bytes,
                     void* stream, void* copy_stream) {
  if (s && s->text_tokens > 0)
    return fail(DIT_ERR_UNSUPPORTED, "dit_serve handles image-only models (text_tokens == 0)");
  dit_status st = check_step_weights(s, w);
  if (st != DIT_OK) return st;
  if (s->patch_in != s->patch_out)
    return fail(DIT_ERR_INVALID_ARG, "the sampler needs patch_in == patch_out (%d != %d)", s->patch_in, s->patch_out);
  if (n_requests < 0 || n_steps < 0) return fail(DIT_ERR_INVALID_ARG, "negative request or step count");
  if (n_requests > 0 && (!reqs || !sigmas)) return fail(DIT_ERR_INVALID_ARG, "reqs or sigmas is NULL");
  if (overlap && !copy_stream) return fail(DIT_ERR_INVALID_ARG, "overlap needs a copy stream");
  if (cw && (!cw->w_t1 || !cw->b_t1 || !cw->w_t2 || !cw->b_t2 || !cw->class_table))
    return fail(DIT_ERR_INVALID_ARG, "a conditioning weight pointer is NULL");
  if (cw && (!aligned(cw->w_t1, 16) || !aligned(cw->w_t2, 16)))
    return fail(DIT_ERR_INVALID_ARG, "w_t1 and w_t2 must be 16-byte aligned");
  for (int i = 0; i < n_requests; ++i) {
    if (!reqs[i].z_in || !reqs[i].z_out) return fail(DIT_ERR_INVALID_ARG, "request %d: z_in or z_out is NULL", i);
    if (cw ? !reqs[i].y : !reqs[i].cond)
      return fail(DIT_ERR_INVALID_ARG, "request %d: %s is NULL", i, cw ? "y" : "cond");
  }
  const Layout L = layout(s, DIT_WS_SERVE);
  if (!workspace || !aligned(workspace, 256)) return fail(DIT_ERR_INVALID_ARG, "workspace NULL or not 256-byte aligned");
  if (ws_bytes < L.total) return fail(DIT_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", ws_bytes, L.total);
  if (n_requests == 0) return DIT_OK;

  hipStream_t hs = (hipStream_t)stream;
  hipStream_t cs = overlap ? (hipStream_t)copy_stream : hs;
  char* ws = (char*)workspace;
  const int B = s->batch, D = s->hidden;
  const size_t zb = (size_t)B * s->tokens * s->patch_out * sizeof(float);
  // ev_in[k]: inputs of the request in slot k are on the device;
  // ev_done[k]: its loop finished; ev_free[k]: its output left the device.
  hipEvent_t ev[6] = {};
  for (hipEvent_t& e : ev) HIP_TRY(hipEventCreateWithFlags(&e, hipEventDisableTiming));
  hipEvent_t *ev_in = ev, *ev_done = ev + 2, *ev_free = ev + 4;
  dit_status result = DIT_OK;
  uint32_t rng = jitter_seed * 2654435761u + 1u;
  auto jitter = [&]() {
    if (!jitter_us) return;
    rng ^= rng << 13; rng ^= rng >> 17; rng ^= rng << 5;  // xorshift32
    std::this_thread::sleep_for(std::chrono::microseconds(rng % (jitter_us + 1)));
  };
  auto fetch = [&](int i) -> hipError_t {  // host -> device slot of request i (on cs)
    const int k = i & 1;
    hipError_t e = hipSuccess;
    if (i >= 2) e = hipStreamWaitEvent(cs, ev_free[k], 0);  // slot's previous output has left
    if (e == hipSuccess) e = hipMemcpyAsync(ws + L.slot_z[k], reqs[i].z_in, zb, hipMemcpyHostToDevice, cs);
    if (e == hipSuccess)
      e = cw ? hipMemcpyAsync(ws + L.slot_y[k], reqs[i].y, (size_t)B * sizeof(int32_t), hipMemcpyHostToDevice, cs)
             : hipMemcpyAsync(ws + L.slot_c[k], reqs[i].cond, (size_t)B * D * sizeof(float), hipMemcpyHostToDevice, cs);
    if (e == hipSuccess) e = hipEventRecord(ev_in[k], cs);
    return e;
  };
  hipError_t e = fetch(0);
  for (int i = 0; i < n_requests && e == hipSuccess && result == DIT_OK; ++i) {
    const int k = i & 1;
    jitter();
    e = hipStreamWaitEvent(hs, ev_in[k], 0);
    if (e != hipSuccess) break;
    result = run_sample_loop(s, w, cw, (const int32_t*)(ws + L.slot_y[k]), (const float*)(ws + L.slot_c[k]), sigmas,
                             n_steps, t_scale, (float*)(ws + L.slot_z[k]), nullptr, L, ws, hs);
    if (result != DIT_OK) break;
    e = hipEventRecord(ev_done[k], hs);
    if (e == hipSuccess && i + 1 < n_requests) e = fetch(i + 1);  // next input moves while request i computes
    if (e == hipSuccess) e = hipStreamWaitEvent(cs, ev_done[k], 0);
    if (e == hipSuccess) e = hipMemcpyAsync(reqs[i].z_out, ws + L.slot_z[k], zb, hipMemcpyDeviceToHost, cs);
    if (e == hipSuccess) e = hipEventRecord(ev_free[k], cs);
  }
  // the caller's stream waits for the last copies; the events can then go
  if (e == hipSuccess && result == DIT_OK && overlap) e = hipStreamWaitEvent(hs, ev_free[(n_requests - 1) & 1], 0);
  for (hipEvent_t& x : ev) (void)hipEventDestroy(x);
  if (result != DIT_OK) return result;
  if (e != hipSuccess) return fail(DIT_ERR_HIP, "dit_serve: %s", hipGetErrorString(e));
  return DIT_OK;
}

dit_status dit_sample_euler(const dit_shape* s, const dit_step_weights* w, const dit_cond_weights* cw,
                            const int32_t* y, const float* cond, const float* sigmas, int32_t n_steps,
                            float t_scale, float* z, const float* x_txt, void* workspace, size_t ws_bytes,
                            void* stream) {
  dit_status st = check_step_weights(s, w);
  if (st != DIT_OK) return st;
  const bool joint = s->text_tokens > 0;
  if (s->patch_in != s->patch_out)
    return fail(DIT_ERR_INVALID_ARG, "the sampler needs patch_in == patch_out (%d != %d)", s->patch_in, s->patch_out);
  if (n_steps < 0) return fail(DIT_ERR_INVALID_ARG, "n_steps %d < 0", n_steps);
  if (!sigmas) return fail(DIT_ERR_INVALID_ARG, "sigmas is NULL");
  if (!z || !aligned(z, 16)) return fail(DIT_ERR_INVALID_ARG, "z NULL or not 16-byte aligned");
  if (joint && (!x_txt || !aligned(x_txt, 16))) return fail(DIT_ERR_INVALID_ARG, "x_txt NULL or not 16-byte aligned");
  if (!joint && x_txt) return fail(DIT_ERR_INVALID_ARG, "x_txt must be NULL when text_tokens == 0");
  if (cw) {
    if (!y || !cw->w_t1 || !cw->b_t1 || !cw->w_t2 || !cw->b_t2 || !cw->class_table)
      return fail(DIT_ERR_INVALID_ARG, "a conditioning pointer (or y) is NULL");
    if (!aligned(cw->w_t1, 16) || !aligned(cw->w_t2, 16))
      return fail(DIT_ERR_INVALID_ARG, "w_t1 and w_t2 must be 16-byte aligned");
  } else if (!cond || !aligned(cond, 4)) {
    return fail(DIT_ERR_INVALID_ARG, "cond NULL or misaligned (and no conditioning weights)");
  }
  const Layout L = layout(s, DIT_WS_SAMPLE);
  if (!workspace || !aligned(workspace, 256)) return fail(DIT_ERR_INVALID_ARG, "workspace NULL or not 256-byte aligned");
  if (ws_bytes < L.total) return fail(DIT_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", ws_bytes, L.total);

  return run_sample_loop(s, w, cw, y, cond, sigmas, n_steps, t_scale, z, x_txt, L, (char*)workspace,
                         (hipStream_t)stream);
}

dit_status dit_cond_embed(const dit_shape* s, const float* t, const int32_t* y, const void* w_t1, const void* b_t1,
                          const void* w_t2, const void* b_t2, const void* class_table, float* cond, void* workspace,
                          size_t ws_bytes, void* stream) {
  dit_status st = check_shape(s, false);
  if (st != DIT_OK) return st;
  if (!t || !y || !w_t1 || !b_t1 || !w_t2 || !b_t2 || !class_table || !cond)
    return fail(DIT_ERR_INVALID_ARG, "a conditioning pointer is NULL");
  if (!aligned(w_t1, 16) || !aligned(w_t2, 16))
    return fail(DIT_ERR_INVALID_ARG, "w_t1 and w_t2 must be 16-byte aligned");
  const Layout L = layout(s, DIT_WS_COND);
  if (!workspace || !aligned(workspace, 256)) return fail(DIT_ERR_INVALID_ARG, "workspace NULL or not 256-byte aligned");
  if (ws_bytes < L.total) return fail(DIT_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", ws_bytes, L.total);
  hipStream_t hs = (hipStream_t)stream;
  char* ws = (char*)workspace;
  HIP_TRY(timed(DIT_K_OTHER, 0, 0, hs, [&]() {
    return launch_cond_embed(s->batch, s->hidden, t, y, w_t1, b_t1, w_t2, b_t2, class_table, (float*)(ws + L.feat),
                             (float*)(ws + L.h1), cond, s->dtype, hs);
  }));
  return DIT_OK;
}

dit_status dit_pos_embed_2d(int32_t grid_h, int32_t grid_w, int32_t hidden, float* pos, void* stream) {
  if (grid_h < 1 || grid_w < 1 || hidden < 4 || hidden % 4 != 0)
    return fail(DIT_ERR_INVALID_ARG, "grid (%d x %d) must be >= 1 and hidden (%d) a positive multiple of 4", grid_h,
                grid_w, hidden);
  if ((long)grid_h * grid_w * hidden >= (1L << 31)) return fail(DIT_ERR_UNSUPPORTED, "position table too large");
  if (!pos || !aligned(pos, 4)) return fail(DIT_ERR_INVALID_ARG, "pos NULL or misaligned");
  HIP_TRY(launch_pos_embed_2d(grid_h, grid_w, hidden, pos, (hipStream_t)stream));
  return DIT_OK;
}

dit_status dit_timing_enable(int kclass, int max_launches) {
  if (kclass < 0 || kclass >= DIT_K_COUNT || max_launches < 1 || max_launches > (1 << 20))
    return fail(DIT_ERR_INVALID_ARG, "bad timing class %d or launch count %d", kclass, max_launches);
  dit_timing_disable();
  std::lock_guard<std::mutex> lk(g_timing.mu);
  g_timing.ev.assign(2 * (size_t)max_launches, nullptr);
  // Timing-only events: without the system-scope fence an event record does
  // not write back and invalidate the L2s, which would add several
  // microseconds per record and slow the bracketed kernel's first accesses.
  for (auto& e : g_timing.ev) {
    hipError_t r = hipEventCreateWithFlags(&e, hipEventDisableSystemFence);
    if (r != hipSuccess) {
      for (auto& f : g_timing.ev)
        if (f) hipEventDestroy(f);
      g_timing.ev.clear();
      return fail(DIT_ERR_HIP, "hipEventCreateWithFlags: %s", hipGetErrorString(r));
    }
  }
  g_timing.kclass = kclass;
  g_timing.max = max_launches;
  g_timing.used = 0;
  g_timing.flops = g_timing.bytes = 0;
  return DIT_OK;
}

dit_status dit_timing_read(double* total_ms, int* launches, double* flops, double* bytes) {
  std::lock_guard<std::mutex> lk(g_timing.mu);
  double ms = 0;
  for (int i = 0; i < g_timing.used; ++i) {
    hipError_t r = hipEventSynchronize(g_timing.ev[2 * i + 1]);
    if (r != hipSuccess) return fail(DIT_ERR_HIP, "hipEventSynchronize: %s", hipGetErrorString(r));
    float t = 0;
    r = hipEventElapsedTime(&t, g_timing.ev[2 * i], g_timing.ev[2 * i + 1]);
    if (r != hipSuccess) return fail(DIT_ERR_HIP, "hipEventElapsedTime: %s", hipGetErrorString(r));
    ms += t;
  }
  if (total_ms) *total_ms = ms;
  if (launches) *launches = g_timing.used;
  if (flops) *flops = g_timing.flops;
  if (bytes) *bytes = g_timing.bytes;
  return DIT_OK;
}

dit_status dit_timing_disable(void) {
  std::lock_guard<std::mutex> lk(g_timing.mu);
  for (auto& e : g_timing.ev)
    if (e) hipEventDestroy(e);
  g_timing.ev.clear();
  g_timing.kclass = -1;
  g_timing.max = g_timing.used = 0;
  return DIT_OK;
}

}  // extern "C"
