// Host side of libkbest: argument validation, launch planning, workspace
// layout and the C entry points declared in include/kbest.h.
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <string>

#include "kbest.h"
#include "kbest_standin.h"
#include "kb_launch.hpp"

namespace kb {
hipError_t launch_k1_reg_bf16_L256(int kc, dim3 grid, const K1Args& a, hipStream_t st);
hipError_t launch_k1_reg_bf16_L128(int kc, dim3 grid, const K1Args& a, hipStream_t st);
hipError_t launch_k1_reg_bf16_L32(int kc, dim3 grid, const K1Args& a, hipStream_t st);
hipError_t launch_k1_reg_f32_L256(int kc, dim3 grid, const K1Args& a, hipStream_t st);
hipError_t launch_k1_reg_f32_L128(int kc, dim3 grid, const K1Args& a, hipStream_t st);
hipError_t launch_k1_reg_f32_L32(int kc, dim3 grid, const K1Args& a, hipStream_t st);
hipError_t launch_k1_dma_L256(int kc, dim3 grid, const K1Args& a, hipStream_t st);
hipError_t launch_k1_dma_L128(int kc, dim3 grid, const K1Args& a, hipStream_t st);
hipError_t launch_k1_dma_L32(int kc, dim3 grid, const K1Args& a, hipStream_t st);
hipError_t launch_k1_reg_bf16_L32M(int kc, dim3 grid, const K1Args& a, hipStream_t st);
hipError_t launch_k1_reg_bf16_L32S(int kc, dim3 grid, const K1Args& a, hipStream_t st);
hipError_t launch_k1_reg_f32_L32M(int kc, dim3 grid, const K1Args& a, hipStream_t st);
hipError_t launch_k1_reg_f32_L32S(int kc, dim3 grid, const K1Args& a, hipStream_t st);
hipError_t launch_k1_dma_L32M(int kc, dim3 grid, const K1Args& a, hipStream_t st);
hipError_t launch_k1_dma_L32S(int kc, dim3 grid, const K1Args& a, hipStream_t st);
hipError_t launch_k1_wide(int kc, dim3 grid, const K1Args& a, hipStream_t st);
hipError_t launch_k1_dma_f32_L256(int kc, dim3 grid, const K1Args& a, hipStream_t st);
hipError_t launch_k1_dma_f32_L128(int kc, dim3 grid, const K1Args& a, hipStream_t st);
hipError_t launch_k1_dma_f32_L32(int kc, dim3 grid, const K1Args& a, hipStream_t st);
hipError_t launch_k1_dma_f32_L32M(int kc, dim3 grid, const K1Args& a, hipStream_t st);
hipError_t launch_k1_dma_f32_L32S(int kc, dim3 grid, const K1Args& a, hipStream_t st);
hipError_t launch_k1_dma_L64(int kc, dim3 grid, const K1Args& a, hipStream_t st);
hipError_t launch_k1_dma_f32_L64(int kc, dim3 grid, const K1Args& a, hipStream_t st);

hipError_t launch_k1(int bf16, int dma, int layout, int kc, dim3 grid, const K1Args& a, hipStream_t st) {
  if (dma && !bf16) {
    switch (layout) {
      case K1_L256: return launch_k1_dma_f32_L256(kc, grid, a, st);
      case K1_L128: return launch_k1_dma_f32_L128(kc, grid, a, st);
      case K1_L32M: return launch_k1_dma_f32_L32M(kc, grid, a, st);
      case K1_L32S: return launch_k1_dma_f32_L32S(kc, grid, a, st);
      case K1_L32: return launch_k1_dma_f32_L32(kc, grid, a, st);
      case K1_L64: return launch_k1_dma_f32_L64(kc, grid, a, st);
      default: return hipErrorInvalidValue;  // the 256 x 256 tile is bf16 only
    }
  }
  if (dma) {
    switch (layout) {
      case K1_W256: return launch_k1_wide(kc, grid, a, st);
      case K1_L256: return launch_k1_dma_L256(kc, grid, a, st);
      case K1_L128: return launch_k1_dma_L128(kc, grid, a, st);
      case K1_L32M: return launch_k1_dma_L32M(kc, grid, a, st);
      case K1_L32S: return launch_k1_dma_L32S(kc, grid, a, st);
      case K1_L64: return launch_k1_dma_L64(kc, grid, a, st);
      default: return launch_k1_dma_L32(kc, grid, a, st);
    }
  }
  if (bf16) {
    switch (layout) {
      case K1_L256: return launch_k1_reg_bf16_L256(kc, grid, a, st);
      case K1_L128: return launch_k1_reg_bf16_L128(kc, grid, a, st);
      case K1_L32M: return launch_k1_reg_bf16_L32M(kc, grid, a, st);
      case K1_L32S: return launch_k1_reg_bf16_L32S(kc, grid, a, st);
      default: return launch_k1_reg_bf16_L32(kc, grid, a, st);
    }
  }
  switch (layout) {
    case K1_L256: return launch_k1_reg_f32_L256(kc, grid, a, st);
    case K1_L128: return launch_k1_reg_f32_L128(kc, grid, a, st);
    case K1_L32M: return launch_k1_reg_f32_L32M(kc, grid, a, st);
    case K1_L32S: return launch_k1_reg_f32_L32S(kc, grid, a, st);
    default: return launch_k1_reg_f32_L32(kc, grid, a, st);
  }
}
}  // namespace kb

namespace {

thread_local std::string g_last_error;

kb_status fail(kb_status status, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
kb_status fail(kb_status status, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return status;
}

kb_status ok() {
  g_last_error.clear();
  return KB_OK;
}

// The projection is planned for MI355X: 256 compute units, one fused
// workgroup per CU (its LDS and registers allow no more).
constexpr int kTargetCUs = 256;

struct Plan {
  int layout, kc, BH, BV;
  int row_tiles, n_vtiles, P, tps;
  size_t stats_off, lists_off, gthr_off, gmax_off, bytes;
};

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Splits whose running row maxima the 256 x 256 tile kernel shares (16 keys per row).
constexpr int kGmaxSplits = 16;

// The wide kernel's W source offsets assume at least one full 256-word tile.
constexpr int kWideMinCols = 256;

// Shapes the DMA pipeline accepts, pointer alignment aside: 64 bytes of an h
// row per stage and whole 4-stage tiles (bf16 H % 128, float32 H % 64), W
// rows of whole 16-byte chunks.
bool dma_shape(int dtype, int H, int V) {
  return dtype == KB_BF16 ? (H % 128 == 0 && V % 8 == 0) : (H % 64 == 0 && V % 4 == 0);
}

// The few-row kernel holds every row's state in LDS next to its partial sums.
constexpr size_t kFewLdsMax = 160 * 1024;
// It streams W at 3.5-4 TB/s and adds its arithmetic after the loads, while
// the matrix-core kernels carry about 20 us of fixed cost per step.  Measured
// per step, both ways, at 1-8 rows: float32 (H 512-1024, V 30k, up to 234 M
// row-weight products) it is 25-40% faster everywhere; bf16 it is faster at
// V=50k, H=1024 up to 4 rows (195 M products; 32-36 against 32-37 us) and
// slower from 6 rows, at V=90k (from one row: 47 against 41 us) and at
// H=2048 (W of 88-102 M weights, where its bf16 dot products are the bound).
constexpr long long kFewMaxWorkF32 = 1ll << 30;

// Tile choice by a cost model.  A step's projection takes about
//   (a H + e) x (rows x words one workgroup covers) x slots + f  microseconds,
// the workgroup covering row tile x word tile x tiles per split, slots = 2
// for a tile planned at two workgroups per CU whose grid exceeds one per CU.  a, e and f
// per layout are fitted by tune_planner.py to the projection times of every
// layout forced in turn (KB_TILE; k = 5) over 40-1280 rows (bf16 2560), one
// table per path: float32 register-staged and float32 on the DMA pipeline at
// H 256-2048 (register-staged: measured while those shapes took that path;
// now H not a multiple of 64), V 8k-60k (120 shapes each), bf16 on the DMA
// pipeline at H 512-2048, V 8k-90k (132 shapes).  Choosing by the model comes
// within 6%, 2% and 9% of the fastest measured layout on each shape.  For
// register-staged float32 the 256-row x 128-word tile is left out: it fits
// the model poorly and was the fastest only by 3-6%, at 160 rows.
struct TileCost {
  int layout, BH, BV;
  double a, e, f;
};
constexpr TileCost kF32Costs[] = {
    {kb::K1_L128, 128, 256, 4.7971e-06, 5.1433e-04, 13.625},
    {kb::K1_L32, 32, 512, 6.7494e-06, 4.2968e-04, 16.657},
    {kb::K1_L32M, 32, 256, 6.7685e-06, 6.3867e-04, 18.986},
    {kb::K1_L32S, 32, 128, 7.6774e-06, 8.7361e-04, 18.167},
};
constexpr TileCost kBf16DmaCosts[] = {
    {kb::K1_W256, 256, 256, 3.1048e-07, 2.2403e-04, 15.484},
    {kb::K1_L128, 128, 256, 4.9823e-07, 3.4975e-04, 18.980},
    {kb::K1_L256, 256, 128, 4.8626e-07, 3.4485e-04, 17.401},
    {kb::K1_L32, 32, 512, 9.8166e-07, 3.7969e-04, 17.161},
    {kb::K1_L32M, 32, 256, 1.2685e-06, 5.1027e-04, 20.342},
    {kb::K1_L32S, 32, 128, 1.4177e-06, 3.1844e-04, 18.122},
    {kb::K1_L64, 64, 128, 7.7745e-07, 2.1370e-04, 17.918},
};
// float32 on the DMA pipeline (fp32 MFMA, operands straight from LDS)
constexpr TileCost kF32DmaCosts[] = {
    {kb::K1_L128, 128, 256, 3.6907e-06, 4.3125e-04, 15.592},
    {kb::K1_L256, 256, 128, 3.7159e-06, 4.2437e-04, 14.462},
    {kb::K1_L32, 32, 512, 4.4843e-06, 5.1425e-04, 15.031},
    {kb::K1_L32M, 32, 256, 4.9426e-06, 6.6724e-04, 18.698},
    {kb::K1_L32S, 32, 128, 4.6148e-06, 5.8893e-04, 18.438},
    {kb::K1_L64, 64, 128, 4.1449e-06, 2.7480e-04, 17.195},
};

// k rounded up to the k-list lengths the projection kernels are built for
int kc_of(int k) { return k <= 4 ? 4 : (k <= 8 ? 8 : (k <= 12 ? 12 : 16)); }

// Workgroups of a layout that one CU holds at once.  On the DMA pipeline the
// 32 x 128 tile (60 KB of LDS, at most 220 registers per lane) and, with
// k <= 8, the 64 x 128 tile (67 KB, built for at most 256 registers) run two
// side by side, one's epilogue and barrier waits overlapping the other's
// products (their grids may reach 512 workgroups); every other tile, and the
// 64 x 128 one with longer lists, fills a CU.
int per_cu(int layout, bool dma, int kc) {
  if (!dma) return 1;
  return layout == kb::K1_L32S || (layout == kb::K1_L64 && kc <= 8) ? 2 : 1;
}

// splits of the vocabulary for a layout: per_cu workgroups per CU over the row tiles
int splits_for(int row_tiles, int n_vtiles, int per) {
  int P = per * kTargetCUs / (row_tiles > 0 ? row_tiles : 1);
  if (P < 1) P = 1;
  if (P > n_vtiles) P = n_vtiles;
  if (P > 256) P = 256;
  return P;
}

// the layout of the least modelled time among n (ties keep the earlier)
template <size_t n>
void pick_by_model(const TileCost (&costs)[n], int N, int H, int V, bool dma, int kc, Plan& p) {
  double best = -1.0;
  for (const TileCost& c : costs) {
    if (c.layout == kb::K1_W256 && V < kWideMinCols) continue;
    if (c.layout == kb::K1_L64 && kc > 8) continue;  // fitted at two workgroups per CU
    const int rt = (N + c.BH - 1) / c.BH, nt = (V + c.BV - 1) / c.BV;
    const int per = per_cu(c.layout, dma, kc);
    const int P = splits_for(rt, nt, per), tps = (nt + P - 1) / P;
    const bool paired = rt * ((nt + tps - 1) / tps) > kTargetCUs;
    // a two-per-CU tile alone on its CU with several tiles to run in turn
    // (one row tile: splits are capped at 256) is slower than the fit says
    // (V=50k, 40 rows, bf16: 64 x 128 measured 43.6 us against 37.5 for
    // 32 x 512); the fit holds for co-resident pairs and single tiles
    if (per == 2 && !paired && tps > 1) continue;
    // a CU that holds two workgroups runs both: twice the words at the
    // co-resident rate (the fit's), once the grid exceeds one per CU
    const int slots = per == 2 && paired ? 2 : 1;
    const double t = (c.a * H + c.e) * (double)c.BH * c.BV * tps * slots + c.f;
    if (best < 0.0 || t < best) {
      best = t;
      p.layout = c.layout;
      p.BH = c.BH;
      p.BV = c.BV;
    }
  }
}
constexpr long long kFewMaxWorkBf16 = 200ll << 20;
constexpr long long kFewMaxWeightsBf16 = 64ll << 20;

// KB_TILE=<rows>x<words> (e.g. 32x256) at call time replaces the modelled
// choice by that tile where the step's path has it (for measuring the cost
// model; the tuning script sets it): 128x256, 256x128, 32x512, 32x256,
// 32x128, 64x128 on the DMA pipeline (dma), and 256x256 on the bf16 DMA
// pipeline with V >= 256 (wide_ok).  Other values are ignored.
void apply_tile_override(bool dma, bool wide_ok, Plan& p) {
  const char* e = getenv("KB_TILE");
  int r = 0, w = 0;
  char tail = 0;
  if (e == nullptr || sscanf(e, "%dx%d%c", &r, &w, &tail) != 2) return;
  int layout = -1;
  if (r == 256 && w == 256 && wide_ok) layout = kb::K1_W256;
  else if (r == 128 && w == 256) layout = kb::K1_L128;
  else if (r == 256 && w == 128) layout = kb::K1_L256;
  else if (r == 32 && w == 512) layout = kb::K1_L32;
  else if (r == 32 && w == 256) layout = kb::K1_L32M;
  else if (r == 32 && w == 128) layout = kb::K1_L32S;
  else if (r == 64 && w == 128 && dma) layout = kb::K1_L64;
  if (layout < 0) return;
  p.layout = layout;
  p.BH = r;
  p.BV = w;
}

Plan make_plan(int dtype, int N, int H, int V, int k, bool dma, bool vec) {
  Plan p{};
  const int few_cw = kb::few_chunk_words(dtype == KB_BF16);
  const int few_nt = (V + few_cw - 1) / few_cw, few_p = std::min(few_nt, kTargetCUs);
  const long long few_work = (long long)N * H * V, few_weights = (long long)H * V;
  const bool few_fits = dtype == KB_BF16 ? (few_work <= kFewMaxWorkBf16 && few_weights <= kFewMaxWeightsBf16)
                                         : few_work <= kFewMaxWorkF32;
  if (vec && N <= kb::FEW_ROWS && V >= few_cw && few_fits &&
      kb::few_lds_needed(dtype == KB_BF16, N, H, (few_nt + few_p - 1) / few_p) <= kFewLdsMax) {
    // a few rows: one pass over W on the vector ALUs; chunks of few_cw words,
    // as many splits as CUs (at most), each a run of whole chunks
    p.layout = kb::K1_FEW;
    p.BH = kb::FEW_ROWS;
    p.BV = few_cw;
  } else if (dma && dma_shape(dtype, H, V)) {
    if (dtype == KB_BF16)
      pick_by_model(kBf16DmaCosts, N, H, V, true, kc_of(k), p);
    else
      pick_by_model(kF32DmaCosts, N, H, V, true, kc_of(k), p);
  } else if (dtype == KB_F32) {
    pick_by_model(kF32Costs, N, H, V, false, kc_of(k), p);
  } else if (N > 192 && dtype == KB_BF16) {
    p.layout = kb::K1_L256;
    p.BH = 256;
    p.BV = 128;
  } else if (N >= 33) {
    p.layout = kb::K1_L128;
    p.BH = 128;
    p.BV = 256;
  } else {
    // 32-row tiles: the word tile sets how many
    // CUs take part.  Of 512, 256 and 128 words, the one with the shortest
    // split (tiles per split x (tile width + a per-tile cost of about 64
    // words' worth)) wins; ties keep the wider tile.
    static const int kLayouts[3] = {kb::K1_L32, kb::K1_L32M, kb::K1_L32S};
    const int rt = (N + 31) / 32;
    long best = -1;
    for (int i = 0; i < 3; ++i) {
      const int bv = 512 >> i;
      const int nt = (V + bv - 1) / bv;
      const int pp = nt < kTargetCUs / rt ? nt : kTargetCUs / rt;
      const long cost = (long)((nt + pp - 1) / pp) * (bv + 64);
      if (best < 0 || cost < best) {
        best = cost;
        p.layout = kLayouts[i];
        p.BV = bv;
      }
    }
    p.BH = 32;
  }
  const bool dma_path = dma && dma_shape(dtype, H, V);
  if (p.layout != kb::K1_FEW) apply_tile_override(dma_path, dtype == KB_BF16 && dma_path && V >= kWideMinCols, p);
  p.kc = kc_of(k);
  p.row_tiles = (N + p.BH - 1) / p.BH;
  p.n_vtiles = (V + p.BV - 1) / p.BV;
  const int P = splits_for(p.row_tiles, p.n_vtiles, per_cu(p.layout, dma_path, p.kc));
  p.tps = (p.n_vtiles + P - 1) / P;
  p.P = (p.n_vtiles + p.tps - 1) / p.tps;  // no empty split
  p.stats_off = 0;
  p.lists_off = align_up((size_t)p.P * N * sizeof(float2), 256);
  p.gthr_off = align_up(p.lists_off + (size_t)p.P * N * k * sizeof(int2), 256);
  p.gmax_off = p.gthr_off + (size_t)p.row_tiles * p.BH * sizeof(uint32_t);  // right after gthr: one reset
  const size_t gmax_n = p.layout == kb::K1_W256 ? (size_t)p.row_tiles * p.BH * kGmaxSplits : 0;
  p.bytes = align_up(p.gmax_off + gmax_n * sizeof(uint32_t), 256);
  return p;
}

// Workspace for a shape: enough for whichever plan the pointers' alignment selects.
size_t workspace_bytes(int dtype, int N, int H, int V, int k) {
  const size_t a = make_plan(dtype, N, H, V, k, true, true).bytes, b = make_plan(dtype, N, H, V, k, false, true).bytes,
               c = make_plan(dtype, N, H, V, k, false, false).bytes;
  return std::max(a, std::max(b, c));
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

kb_status validate_step(int dtype, int N, int H, int V, int k, int S) {
  if (dtype != KB_F32 && dtype != KB_BF16) return fail(KB_ERR_INVALID_ARG, "unknown dtype %d", dtype);
  if (N < 0 || S < 0) return fail(KB_ERR_INVALID_ARG, "negative N (%d) or S (%d)", N, S);
  if ((N == 0) != (S == 0)) return fail(KB_ERR_INVALID_ARG, "N = %d and S = %d: both or neither must be 0", N, S);
  if (H < 1 || V < 1) return fail(KB_ERR_INVALID_ARG, "H = %d and V = %d must be >= 1", H, V);
  if (k < 1 || k > KB_MAX_K || k > V)
    return fail(KB_ERR_INVALID_ARG, "k = %d outside [1, min(%d, V = %d)]", k, KB_MAX_K, V);
  if (N < S) return fail(KB_ERR_INVALID_ARG, "N = %d < S = %d: N >= S is required", N, S);
  if ((long long)N * k > INT_MAX || (long long)S * k > INT_MAX || (long long)H * V > (1LL << 40))
    return fail(KB_ERR_UNSUPPORTED, "shape too large");
  // a sentence's flat candidate index (row - first row) * V + word is an int32
  if ((long long)N * V > INT_MAX) return fail(KB_ERR_UNSUPPORTED, "N * V = %lld exceeds INT_MAX", (long long)N * V);
  // byte offsets into h are 32-bit in the projection kernels
  if ((long long)N * H * (dtype == KB_BF16 ? 2 : 4) >= (1LL << 32)) return fail(KB_ERR_UNSUPPORTED, "h is 4 GiB or larger");
  return KB_OK;
}

// KB_DEBUG=1: validate device-resident index arrays before anything else is
// enqueued.  The verdict word goes to `flag` (an int32 of the call's output
// that the call overwrites when it goes ahead) and is read back after a wait.
bool debug_checks() {
  const char* e = getenv("KB_DEBUG");
  return e != nullptr && e[0] == '1' && e[1] == 0;
}

kb_status debug_verdict(hipError_t e, const int32_t* flag, hipStream_t hs, const char* what) {
  if (e != hipSuccess) return fail(KB_ERR_HIP, "KB_DEBUG check launch: %s", hipGetErrorString(e));
  int32_t v = -1;
  e = hipMemcpyAsync(&v, flag, sizeof v, hipMemcpyDeviceToHost, hs);
  if (e == hipSuccess) e = hipStreamSynchronize(hs);
  if (e != hipSuccess) return fail(KB_ERR_HIP, "KB_DEBUG check read-back: %s", hipGetErrorString(e));
  if (v != 0) return fail(KB_ERR_INVALID_ARG, "KB_DEBUG: %s (check word 0x%x)", what, (unsigned)v);
  return KB_OK;
}

kb_status debug_offsets(int S, int N, const int32_t* off, int32_t* flag, hipStream_t hs) {
  if (!debug_checks()) return KB_OK;
  return debug_verdict(kb::launch_check_offsets(S, N, off, flag, hs), flag, hs,
                       "sent_offsets break 0 = off[0] <= off[1] <= ... <= off[S] <= N");
}

// Whether the operands allow 16-byte vector loads, and the plan they select.
bool vec_operands(int dtype, int H, int V, const void* h, const void* W) {
  const int vec = dtype == KB_BF16 ? 8 : 4;
  return (H % vec == 0) && (V % vec == 0) && aligned(h, 16) && aligned(W, 16);
}
Plan plan_for(int dtype, int N, int H, int V, int k, const void* h, const void* W, const float* b) {
  const bool vec = vec_operands(dtype, H, V, h, W);
  const bool dma = dma_shape(dtype, H, V) && vec && aligned(b, 16);
  return make_plan(dtype, N, H, V, k, dma, vec);
}

// Alignment checks, plan, threshold reset and the projection kernel (K1)
// shared by the k-best step, the greedy argmax and the vocabulary shards.  On
// KB_OK, a1 and p describe the launched projection; its partials are in the
// workspace, or in stats_out / lists_out when given (split rows N apart).
kb_status launch_projection(int dtype, int N, int H, int V, int k, const void* h, const void* W, const float* b,
                      void* ws, size_t ws_bytes, hipStream_t hs, bool no_stats, void* ev0, void* ev1,
                      kb::K1Args& a1, Plan& p, float2* stats_out = nullptr, int2* lists_out = nullptr) {
  const size_t esz = dtype == KB_BF16 ? 2 : 4;
  if (!aligned(h, esz) || !aligned(W, esz) || !aligned(b, 4))
    return fail(KB_ERR_INVALID_ARG, "h, W or b misaligned for its element type");
  const bool vec_ok = vec_operands(dtype, H, V, h, W);
  const bool dma = dma_shape(dtype, H, V) && vec_ok && aligned(b, 16);
  p = make_plan(dtype, N, H, V, k, dma, vec_ok);
  const size_t need = workspace_bytes(dtype, N, H, V, k);
  if (!ws) return fail(KB_ERR_WORKSPACE, "workspace is null (%zu bytes needed)", need);
  if (!aligned(ws, 256)) return fail(KB_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if (ws_bytes < need) return fail(KB_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", ws_bytes, need);
  if (p.P > 256) return fail(KB_ERR_UNSUPPORTED, "too many vocabulary splits");

  a1 = kb::K1Args{};
  a1.h = h;
  a1.W = W;
  a1.b = b;
  a1.N = N;
  a1.H = H;
  a1.V = V;
  a1.k = k;
  a1.tps = p.tps;
  a1.n_vtiles = p.n_vtiles;
  a1.vec_ok = vec_ok;
  a1.stats = stats_out ? stats_out : reinterpret_cast<float2*>((char*)ws + p.stats_off);
  a1.lists = lists_out ? lists_out : reinterpret_cast<int2*>((char*)ws + p.lists_off);
  a1.gthr = reinterpret_cast<uint32_t*>((char*)ws + p.gthr_off);
  a1.gmax = reinterpret_cast<uint32_t*>((char*)ws + p.gmax_off);
  a1.row_tiles = p.row_tiles;
  a1.P = p.P;
  a1.grp = p.row_tiles < 4 ? p.row_tiles : 4;
  a1.no_stats = (no_stats && p.layout == kb::K1_W256 && p.kc == 4) ? 1 : 0;

  // With one tile per split and every workgroup resident from the start, no
  // workgroup reads a threshold before the others publish theirs: the other
  // tiles' kernels then share none, and the reset is not needed.
  const bool all_resident = p.P * p.row_tiles <= per_cu(p.layout, dma, p.kc) * kTargetCUs;
  a1.share = (p.layout == kb::K1_W256 || p.tps > 1 || !all_resident) ? 1 : 0;
  hipError_t e = hipSuccess;
  if (p.layout != kb::K1_FEW && a1.share) {  // the few-row kernel shares no thresholds
    const int n_zero = p.row_tiles * p.BH * (p.layout == kb::K1_W256 ? 1 + kGmaxSplits : 1);  // gthr (+ gmax)
    e = kb::launch_zero_u32(a1.gthr, n_zero, hs);
    if (e != hipSuccess) return fail(KB_ERR_HIP, "threshold reset kernel launch: %s", hipGetErrorString(e));
  }
  if (ev0) {
    e = hipEventRecord(reinterpret_cast<hipEvent_t>(ev0), hs);
    if (e != hipSuccess) return fail(KB_ERR_HIP, "hipEventRecord: %s", hipGetErrorString(e));
  }
  if (p.layout == kb::K1_FEW)
    e = kb::launch_k1_few(dtype == KB_BF16, dim3(p.P), a1, hs);
  else
    e = kb::launch_k1(dtype == KB_BF16, dma, p.layout, p.kc, dim3(p.P * p.row_tiles), a1, hs);
  if (e != hipSuccess) return fail(KB_ERR_HIP, "projection kernel launch: %s", hipGetErrorString(e));
  if (ev1) {
    e = hipEventRecord(reinterpret_cast<hipEvent_t>(ev1), hs);
    if (e != hipSuccess) return fail(KB_ERR_HIP, "hipEventRecord: %s", hipGetErrorString(e));
  }
  return KB_OK;
}

kb_status kbest_step_impl(int dtype, int N, int H, int V, int k, int S, const void* h, const void* W, const float* b,
                    const float* prev, const int32_t* off, int32_t* tok, int32_t* par, float* score,
                    float* row_lse, void* ws, size_t ws_bytes, void* stream, void* ev0, void* ev1) {
  kb_status st = validate_step(dtype, N, H, V, k, S);
  if (st != KB_OK) return st;
  if (N == 0) return ok();
  if (!h || !W || !b || !prev || !off || !tok || !par || !score)
    return fail(KB_ERR_INVALID_ARG, "null input or output pointer");
  if (!aligned(prev, 4)) return fail(KB_ERR_INVALID_ARG, "prev misaligned");
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  if ((st = debug_offsets(S, N, off, tok, hs)) != KB_OK) return st;
  kb::K1Args a1;
  Plan p;
  st = launch_projection(dtype, N, H, V, k, h, W, b, ws, ws_bytes, hs, false, ev0, ev1, a1, p);
  if (st != KB_OK) return st;

  kb::K2Args a2{};
  a2.stats = a1.stats;
  a2.lists = a1.lists;
  a2.P = p.P;
  a2.N = N;
  a2.V = V;
  a2.k = k;
  a2.S = S;
  a2.prev = prev;
  a2.off = off;
  a2.tok = tok;
  a2.par = par;
  a2.score = score;
  a2.row_lse = row_lse;
  hipError_t e = kb::launch_k2(a2, hs);
  if (e != hipSuccess) return fail(KB_ERR_HIP, "merge kernel launch: %s", hipGetErrorString(e));
  return ok();
}

}  // namespace

// ---- the unfused baseline (Algorithm 3; Algorithm 4 over stored scores)
namespace {
struct UfPlan {
  kb::K1Args a1;
  int row_tiles, P;
  size_t logits_off, stats_off, lists_off, gthr_off, bytes;
};

bool uf_shape(int dtype, int H, int V) { return dtype == KB_BF16 && dma_shape(dtype, H, V) && V >= kWideMinCols; }

UfPlan uf_plan(int N, int H, int V, int k) {
  UfPlan u{};
  u.row_tiles = (N + 255) / 256;
  const int n_vtiles = (V + 255) / 256;
  int P = kTargetCUs / u.row_tiles;
  if (P < 1) P = 1;
  if (P > n_vtiles) P = n_vtiles;
  const int tps = (n_vtiles + P - 1) / P;
  u.P = (n_vtiles + tps - 1) / tps;
  u.logits_off = 0;
  u.stats_off = align_up((size_t)N * V * sizeof(float), 256);
  u.lists_off = align_up(u.stats_off + (size_t)N * sizeof(float2), 256);
  u.gthr_off = align_up(u.lists_off + (size_t)N * k * sizeof(int2), 256);
  u.bytes = align_up(u.gthr_off + (size_t)u.row_tiles * 256 * sizeof(uint32_t), 256);
  u.a1.N = N;
  u.a1.H = H;
  u.a1.V = V;
  u.a1.k = k;
  u.a1.tps = tps;
  u.a1.n_vtiles = n_vtiles;
  u.a1.vec_ok = 1;
  u.a1.row_tiles = u.row_tiles;
  u.a1.P = u.P;
  u.a1.grp = u.row_tiles < 4 ? u.row_tiles : 4;
  return u;
}

kb_status record(void* const* ev, int n_ev, int i, hipStream_t hs) {
  if (!ev || i >= n_ev || !ev[i]) return KB_OK;
  hipError_t e = hipEventRecord(reinterpret_cast<hipEvent_t>(ev[i]), hs);
  return e == hipSuccess ? KB_OK : fail(KB_ERR_HIP, "hipEventRecord: %s", hipGetErrorString(e));
}
}  // namespace

extern "C" {

int kb_abi_version(void) { return KB_ABI_VERSION; }

const char* kb_status_string(kb_status s) {
  switch (s) {
    case KB_OK: return "ok";
    case KB_ERR_INVALID_ARG: return "invalid argument";
    case KB_ERR_UNSUPPORTED: return "unsupported";
    case KB_ERR_WORKSPACE: return "workspace missing or too small";
    case KB_ERR_HIP: return "HIP error";
    default: return "unknown status";
  }
}

const char* kb_last_error(void) { return g_last_error.c_str(); }

kb_status kb_kbest_plan(int dtype, int N, int H, int V, int k, const void* h, const void* W, const float* b,
                        int32_t* plan_out) {
  if (!plan_out) return fail(KB_ERR_INVALID_ARG, "plan_out is null");
  kb_status st = validate_step(dtype, N, H, V, k, N > 0 ? 1 : 0);
  if (st != KB_OK) return st;
  for (int i = 0; i < KB_PLAN_FIELDS; ++i) plan_out[i] = 0;
  if (N == 0) return ok();
  const size_t esz = dtype == KB_BF16 ? 2 : 4;
  if (!aligned(h, esz) || !aligned(W, esz) || !aligned(b, 4))
    return fail(KB_ERR_INVALID_ARG, "h, W or b misaligned for its element type");
  const bool vec = vec_operands(dtype, H, V, h, W);
  const bool dma = dma_shape(dtype, H, V) && vec && aligned(b, 16);
  const Plan p = make_plan(dtype, N, H, V, k, dma, vec);
  plan_out[KB_PLAN_KERNEL] = p.layout == kb::K1_FEW ? KB_KERNEL_FEW
                             : p.layout == kb::K1_W256 ? KB_KERNEL_WIDE
                             : dma ? KB_KERNEL_DMA : KB_KERNEL_REG;
  plan_out[KB_PLAN_TILE_ROWS] = p.BH;
  plan_out[KB_PLAN_TILE_WORDS] = p.BV;
  plan_out[KB_PLAN_ROW_TILES] = p.row_tiles;
  plan_out[KB_PLAN_SPLITS] = p.P;
  plan_out[KB_PLAN_TILES_PER_SPLIT] = p.tps;
  return ok();
}

size_t kb_kbest_workspace_bytes(int dtype, int N, int H, int V, int k, int S) {
  if (validate_step(dtype, N, H, V, k, S) != KB_OK || N == 0) return 0;
  return workspace_bytes(dtype, N, H, V, k);
}

kb_status kb_kbest_step(int dtype, int N, int H, int V, int k, int S, const void* h, const void* W, const float* b,
                  const float* prev_score, const int32_t* sent_offsets, int32_t* out_token, int32_t* out_parent,
                  float* out_score, float* out_row_lse, void* workspace, size_t workspace_bytes, void* stream) {
  return kbest_step_impl(dtype, N, H, V, k, S, h, W, b, prev_score, sent_offsets, out_token, out_parent,
                         out_score, out_row_lse, workspace, workspace_bytes, stream, nullptr, nullptr);
}

kb_status kb_kbest_step_events(int dtype, int N, int H, int V, int k, int S, const void* h, const void* W,
                         const float* b, const float* prev_score, const int32_t* sent_offsets, int32_t* out_token,
                         int32_t* out_parent, float* out_score, float* out_row_lse, void* workspace,
                         size_t workspace_bytes, void* stream, void* proj_begin_event, void* proj_end_event) {
  return kbest_step_impl(dtype, N, H, V, k, S, h, W, b, prev_score, sent_offsets, out_token, out_parent,
                         out_score, out_row_lse, workspace, workspace_bytes, stream, proj_begin_event,
                         proj_end_event);
}

// ---- the step without a caller workspace: the projection's partials and
// shared thresholds go to a fixed device array of this library instead
}  // extern "C"

namespace {
constexpr size_t kScratchBytes = (size_t)16 << 20;
constexpr int kMaxDevices = 64;
// One copy per device, held from module load until the process ends.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

// Device address of `scratch` on the current device, looked up once per
// device (the array's name is a host-side stand-in, not a device address).
kb_status scratch_ptr(void** out) {
  static std::mutex mu;
  static void* ptrs[kMaxDevices] = {};
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(KB_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(KB_ERR_UNSUPPORTED, "device %d beyond %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(mu);
  if (ptrs[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr)
      return fail(KB_ERR_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    ptrs[dev] = p;
  }
  *out = ptrs[dev];
  return KB_OK;
}
}  // namespace

extern "C" {

size_t kb_kbest_step_scratch_max(void) { return kScratchBytes; }

kb_status kb_kbest_step_noalloc(int dtype, int N, int H, int V, int k, int S, const void* h, const void* W,
                                const float* b, const float* prev_score, const int32_t* sent_offsets,
                                int32_t* out_token, int32_t* out_parent, float* out_score, float* out_row_lse,
                                void* stream) {
  kb_status st = validate_step(dtype, N, H, V, k, S);
  if (st != KB_OK) return st;
  if (N == 0) return ok();
  const size_t need = workspace_bytes(dtype, N, H, V, k);
  if (need > kScratchBytes)
    return fail(KB_ERR_UNSUPPORTED, "this shape needs %zu bytes of scratch; the fixed array holds %zu", need,
                kScratchBytes);
  void* ws = nullptr;
  if ((st = scratch_ptr(&ws)) != KB_OK) return st;
  return kbest_step_impl(dtype, N, H, V, k, S, h, W, b, prev_score, sent_offsets, out_token, out_parent, out_score,
                         out_row_lse, ws, kScratchBytes, stream, nullptr, nullptr);
}


size_t kb_unfused_workspace_bytes(int dtype, int N, int H, int V, int k, int S) {
  if (validate_step(dtype, N, H, V, k, S) != KB_OK || N == 0 || !uf_shape(dtype, H, V)) return 0;
  return uf_plan(N, H, V, k).bytes;
}

kb_status kb_kbest_step_unfused(int mode, int dtype, int N, int H, int V, int k, int S, const void* h, const void* W,
                          const float* b, const float* prev_score, const int32_t* sent_offsets, int32_t* out_token,
                          int32_t* out_parent, float* out_score, float* out_row_lse, void* workspace,
                          size_t workspace_bytes, void* const* stage_events, int n_events, void* stream) {
  if (mode != 0 && mode != 1) return fail(KB_ERR_INVALID_ARG, "mode %d: 0 (Algorithm 3) or 1 (Algorithm 4)", mode);
  kb_status st = validate_step(dtype, N, H, V, k, S);
  if (st != KB_OK) return st;
  if (N == 0) return ok();
  if (!uf_shape(dtype, H, V))
    return fail(KB_ERR_UNSUPPORTED, "the unfused baseline needs bf16, H %% 128 == 0, V %% 8 == 0 and V >= 256");
  if (!h || !W || !b || !prev_score || !sent_offsets || !out_token || !out_parent || !out_score)
    return fail(KB_ERR_INVALID_ARG, "null input or output pointer");
  if (!aligned(h, 16) || !aligned(W, 16) || !aligned(b, 16) || !aligned(prev_score, 4))
    return fail(KB_ERR_INVALID_ARG, "h, W and b must be 16-byte aligned, prev 4-byte aligned");
  UfPlan u = uf_plan(N, H, V, k);
  if (!workspace) return fail(KB_ERR_WORKSPACE, "workspace is null (%zu bytes needed)", u.bytes);
  if (!aligned(workspace, 256)) return fail(KB_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if (workspace_bytes < u.bytes) return fail(KB_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", workspace_bytes, u.bytes);
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  if ((st = debug_offsets(S, N, sent_offsets, out_token, hs)) != KB_OK) return st;
  char* ws = static_cast<char*>(workspace);
  float* x = reinterpret_cast<float*>(ws + u.logits_off);
  float2* stats = reinterpret_cast<float2*>(ws + u.stats_off);
  int2* lists = reinterpret_cast<int2*>(ws + u.lists_off);
  u.a1.h = h;
  u.a1.W = W;
  u.a1.b = b;
  u.a1.logits = x;
  u.a1.gthr = reinterpret_cast<uint32_t*>(ws + u.gthr_off);  // read by the kernel's pipeline, not used
  u.a1.gmax = u.a1.gthr;
  u.a1.stats = stats;
  u.a1.lists = lists;
  hipError_t e;
#define UF_CHECK(call, what)                                                   \
  do {                                                                         \
    e = (call);                                                                \
    if (e != hipSuccess) return fail(KB_ERR_HIP, what ": %s", hipGetErrorString(e)); \
  } while (0)
  if ((st = record(stage_events, n_events, 0, hs)) != KB_OK) return st;
  UF_CHECK(kb::launch_k1_wide_store(dim3(u.P * u.row_tiles), u.a1, hs), "projection kernel launch");
  if ((st = record(stage_events, n_events, 1, hs)) != KB_OK) return st;
  if (mode == 0) {
    UF_CHECK(kb::launch_uf_add_bias(x, b, N, V, hs), "bias kernel launch");
    if ((st = record(stage_events, n_events, 2, hs)) != KB_OK) return st;
    UF_CHECK(kb::launch_uf_softmax3(x, N, V, out_row_lse, hs), "softmax kernel launch");
    if ((st = record(stage_events, n_events, 3, hs)) != KB_OK) return st;
    UF_CHECK(kb::launch_uf_kbest_rows(x, N, V, k, stats, lists, hs), "k-best kernel launch");
  } else {
    UF_CHECK(kb::launch_uf_fused_rows(x, b, N, V, k, stats, lists, hs), "fused pass launch");
  }
  if ((st = record(stage_events, n_events, mode == 0 ? 4 : 2, hs)) != KB_OK) return st;
  kb::K2Args a2{};
  a2.stats = stats;
  a2.lists = lists;
  a2.P = 1;
  a2.N = N;
  a2.V = V;
  a2.k = k;
  a2.S = S;
  a2.prev = prev_score;
  a2.off = sent_offsets;
  a2.tok = out_token;
  a2.par = out_parent;
  a2.score = out_score;
  a2.row_lse = mode == 0 ? nullptr : out_row_lse;  // Algorithm 3's softmax wrote it
  UF_CHECK(kb::launch_k2(a2, hs), "merge kernel launch");
#undef UF_CHECK
  if ((st = record(stage_events, n_events, mode == 0 ? 5 : 3, hs)) != KB_OK) return st;
  return ok();
}

size_t kb_argmax_workspace_bytes(int dtype, int N, int H, int V) {
  if (validate_step(dtype, N, H, V, 1, N > 0 ? 1 : 0) != KB_OK || N == 0) return 0;
  return workspace_bytes(dtype, N, H, V, 1);
}

kb_status kb_argmax_step(int dtype, int N, int H, int V, const void* h, const void* W, const float* b, int32_t* out_token,
                   float* out_logit, void* workspace, size_t workspace_bytes, void* stream) {
  kb_status st = validate_step(dtype, N, H, V, 1, N > 0 ? 1 : 0);
  if (st != KB_OK) return st;
  if (N == 0) return ok();
  if (!h || !W || !b || !out_token || !out_logit) return fail(KB_ERR_INVALID_ARG, "null input or output pointer");
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  kb::K1Args a1;
  Plan p;
  st = launch_projection(dtype, N, H, V, 1, h, W, b, workspace, workspace_bytes, hs, true, nullptr, nullptr, a1, p);
  if (st != KB_OK) return st;
  hipError_t e = kb::launch_k2_argmax(a1.lists, p.P, N, out_token, out_logit, hs);
  if (e != hipSuccess) return fail(KB_ERR_HIP, "argmax merge kernel launch: %s", hipGetErrorString(e));
  return ok();
}

kb_status kb_beam_finish(int S, int k, int t, int T, int eos, const int32_t* token, const int32_t* parent,
                   const float* score, const int32_t* sent_id, int32_t* beam, const int32_t* prev_keep,
                   int prev_hist_base, int hist_base, int32_t* hist_token, int32_t* hist_parent, int32_t* fin_count,
                   float* fin_score, int32_t* fin_len, int32_t* fin_hist, uint8_t* alive, void* stream) {
  if (S < 0 || k < 1 || k > KB_MAX_K || T < 1 || t < 0 || t >= T)
    return fail(KB_ERR_INVALID_ARG, "S = %d, k = %d, t = %d, T = %d", S, k, t, T);
  if (hist_base < 0 || prev_hist_base < 0 || (long long)hist_base + (long long)S * k > INT_MAX)
    return fail(KB_ERR_INVALID_ARG, "history offsets out of range");
  if (S == 0) return ok();
  if (!token || !parent || !score || !sent_id || !beam || !hist_token || !hist_parent || !fin_count || !fin_score ||
      !fin_len || !fin_hist || !alive)
    return fail(KB_ERR_INVALID_ARG, "null pointer");
  hipError_t e = kb::launch_beam_finish(S, k, t, T, eos, token, parent, score, sent_id, beam, prev_keep,
                                        prev_hist_base, hist_base, hist_token, hist_parent, fin_count, fin_score,
                                        fin_len, fin_hist, alive, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(KB_ERR_HIP, "beam finish kernel launch: %s", hipGetErrorString(e));
  return ok();
}

kb_status kb_beam_backtrace(int S0, int k, int T, float alpha, const int32_t* fin_count, const float* fin_score,
                      const int32_t* fin_len, const int32_t* fin_hist, const int32_t* hist_token,
                      const int32_t* hist_parent, int32_t* out_tokens, int32_t* out_len, float* out_score,
                      float* out_norm, void* stream) {
  if (S0 < 0 || k < 1 || k > KB_MAX_K || T < 1) return fail(KB_ERR_INVALID_ARG, "S0 = %d, k = %d, T = %d", S0, k, T);
  if (S0 == 0) return ok();
  if (!fin_count || !fin_score || !fin_len || !fin_hist || !hist_token || !hist_parent || !out_tokens || !out_len ||
      !out_score || !out_norm)
    return fail(KB_ERR_INVALID_ARG, "null pointer");
  hipError_t e = kb::launch_beam_backtrace(S0, k, T, alpha, fin_count, fin_score, fin_len, fin_hist, hist_token,
                                           hist_parent, out_tokens, out_len, out_score, out_norm,
                                           reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(KB_ERR_HIP, "backtrace kernel launch: %s", hipGetErrorString(e));
  return ok();
}

size_t kb_compact_workspace_bytes(int M) { return M > 0 ? kb::compact_entries_ws_bytes(M) : 0; }

kb_status kb_compact_batch(int M, const uint8_t* alive_mask, int32_t* keep_idx, int32_t* kept_count,
                           const int32_t* entry_sentence, int32_t* new_sent_offsets, int32_t* new_S, void* workspace,
                           size_t workspace_bytes, void* stream) {
  if (M < 0) return fail(KB_ERR_INVALID_ARG, "M = %d < 0", M);
  if (!kept_count || (M > 0 && (!alive_mask || !keep_idx)))
    return fail(KB_ERR_INVALID_ARG, "null alive_mask, keep_idx or kept_count");
  if ((new_sent_offsets || new_S) && !entry_sentence && M > 0)
    return fail(KB_ERR_INVALID_ARG, "new_sent_offsets and new_S need entry_sentence");
  const size_t need = kb_compact_workspace_bytes(M);
  if (need > 0) {
    if (!workspace) return fail(KB_ERR_WORKSPACE, "workspace is null (%zu bytes needed)", need);
    if (!aligned(workspace, 4)) return fail(KB_ERR_WORKSPACE, "workspace must be 4-byte aligned");
    if (workspace_bytes < need) return fail(KB_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", workspace_bytes, need);
  }
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  if (entry_sentence && M > 0 && debug_checks()) {
    kb_status st = debug_verdict(kb::launch_check_sorted(M, entry_sentence, kept_count, hs), kept_count, hs,
                                 "entry_sentence must be >= 0 and non-decreasing");
    if (st != KB_OK) return st;
  }
  hipError_t e = kb::launch_compact_entries(M, alive_mask, keep_idx, kept_count, entry_sentence, new_sent_offsets,
                                            new_S, workspace, hs);
  if (e != hipSuccess) return fail(KB_ERR_HIP, "compaction kernel launch: %s", hipGetErrorString(e));
  return ok();
}

kb_status kb_compact_beams(int S, int k, const uint8_t* alive, int32_t* keep_idx, int32_t* kept_count,
                           int32_t* new_sent_offsets, int32_t* kept_sentence, int32_t* new_S, void* stream) {
  if (S < 0) return fail(KB_ERR_INVALID_ARG, "S = %d < 0", S);
  if (k < 1 || k > 1023) return fail(KB_ERR_INVALID_ARG, "k = %d outside [1, 1023]", k);
  if ((long long)S * k > INT_MAX) return fail(KB_ERR_UNSUPPORTED, "S * k too large");
  if (!kept_count || (S > 0 && (!alive || !keep_idx)))
    return fail(KB_ERR_INVALID_ARG, "null alive, keep_idx or kept_count");
  hipError_t e = kb::launch_compact(S, k, alive, keep_idx, kept_count, new_sent_offsets, kept_sentence, new_S,
                                    reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(KB_ERR_HIP, "compaction kernel launch: %s", hipGetErrorString(e));
  return ok();
}

kb_status kb_gather_rows(int n_max, const int32_t* n_dev, const int32_t* idx, const void* src, void* dst,
                   size_t row_bytes, void* stream) {
  if (n_max < 0) return fail(KB_ERR_INVALID_ARG, "n_max = %d < 0", n_max);
  if (row_bytes == 0 || row_bytes % 4 != 0) return fail(KB_ERR_INVALID_ARG, "row_bytes must be a positive multiple of 4");
  if (row_bytes / 4 > INT_MAX) return fail(KB_ERR_UNSUPPORTED, "row too long");
  if (n_max == 0) return ok();
  if (!idx || !src || !dst) return fail(KB_ERR_INVALID_ARG, "null idx, src or dst");
  if (!aligned(src, 4) || !aligned(dst, 4)) return fail(KB_ERR_INVALID_ARG, "src and dst must be 4-byte aligned");
  hipError_t e = kb::launch_gather(n_max, n_dev, idx, src, dst, row_bytes, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(KB_ERR_HIP, "gather kernel launch: %s", hipGetErrorString(e));
  return ok();
}

// ---- vocabulary shards (Algorithm 6 across devices): one GPU's part
kb_status kb_shard_splits(int dtype, int N, int H, int V_shard, int k, const void* h, const void* W_shard,
                    const float* b_shard, int* splits) {
  if (!splits) return fail(KB_ERR_INVALID_ARG, "splits is null");
  kb_status st = validate_step(dtype, N, H, V_shard, k, N > 0 ? 1 : 0);
  if (st != KB_OK) return st;
  if (N == 0) {
    *splits = 0;
    return ok();
  }
  if (!h || !W_shard || !b_shard) return fail(KB_ERR_INVALID_ARG, "null h, W_shard or b_shard");
  *splits = plan_for(dtype, N, H, V_shard, k, h, W_shard, b_shard).P;
  return ok();
}

size_t kb_shard_workspace_bytes(int dtype, int N, int H, int V_shard, int k) {
  if (N <= 0 || H < 1 || V_shard < 1 || k < 1 || k > KB_MAX_K) return 0;
  return workspace_bytes(dtype, N, H, V_shard, k);
}

kb_status kb_shard_partials(int dtype, int N, int H, int V_shard, int word_base, int k, const void* h,
                      const void* W_shard, const float* b_shard, float* stats, int32_t* lists, void* workspace,
                      size_t workspace_bytes, void* stream) {
  kb_status st = validate_step(dtype, N, H, V_shard, k, N > 0 ? 1 : 0);
  if (st != KB_OK) return st;
  if (N == 0) return ok();
  if (!h || !W_shard || !b_shard || !stats || !lists) return fail(KB_ERR_INVALID_ARG, "null input or output pointer");
  if (word_base < 0 || (long long)word_base + V_shard > INT_MAX)
    return fail(KB_ERR_INVALID_ARG, "word_base = %d outside [0, INT_MAX - V_shard]", word_base);
  if (!aligned(stats, 8) || !aligned(lists, 8)) return fail(KB_ERR_INVALID_ARG, "stats and lists must be 8-byte aligned");
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  kb::K1Args a1;
  Plan p;
  st = launch_projection(dtype, N, H, V_shard, k, h, W_shard, b_shard, workspace, workspace_bytes, hs, false, nullptr,
                         nullptr, a1, p, reinterpret_cast<float2*>(stats), reinterpret_cast<int2*>(lists));
  if (st != KB_OK) return st;
  hipError_t e = kb::launch_add_word_base(reinterpret_cast<int2*>(lists), (size_t)p.P * N * k, word_base, V_shard, hs);
  if (e != hipSuccess) return fail(KB_ERR_HIP, "word offset kernel launch: %s", hipGetErrorString(e));
  return ok();
}

kb_status kb_merge_partials(int N, int V, int k, int S, int P, const float* stats, const int32_t* lists,
                      const float* prev_score, const int32_t* sent_offsets, int32_t* out_token, int32_t* out_parent,
                      float* out_score, float* out_row_lse, void* stream) {
  if (N < 0 || S < 0) return fail(KB_ERR_INVALID_ARG, "negative N (%d) or S (%d)", N, S);
  if ((N == 0) != (S == 0)) return fail(KB_ERR_INVALID_ARG, "N = %d and S = %d: both or neither must be 0", N, S);
  if (N < S) return fail(KB_ERR_INVALID_ARG, "N = %d < S = %d: N >= S is required", N, S);
  if (V < 1) return fail(KB_ERR_INVALID_ARG, "V = %d must be >= 1", V);
  if (k < 1 || k > KB_MAX_K || k > V) return fail(KB_ERR_INVALID_ARG, "k = %d outside [1, min(%d, V = %d)]", k, KB_MAX_K, V);
  if (P < 1 || P > 256) return fail(KB_ERR_UNSUPPORTED, "P = %d splits outside [1, 256]", P);
  if ((long long)N * k * P > INT_MAX || (long long)N * V > INT_MAX) return fail(KB_ERR_UNSUPPORTED, "shape too large");
  if (N == 0) return ok();
  if (!stats || !lists || !prev_score || !sent_offsets || !out_token || !out_parent || !out_score)
    return fail(KB_ERR_INVALID_ARG, "null input or output pointer");
  if (!aligned(stats, 8) || !aligned(lists, 8)) return fail(KB_ERR_INVALID_ARG, "stats and lists must be 8-byte aligned");
  kb_status st = debug_offsets(S, N, sent_offsets, out_token, reinterpret_cast<hipStream_t>(stream));
  if (st != KB_OK) return st;
  kb::K2Args a2{};
  a2.stats = reinterpret_cast<const float2*>(stats);
  a2.lists = reinterpret_cast<const int2*>(lists);
  a2.P = P;
  a2.N = N;
  a2.V = V;
  a2.k = k;
  a2.S = S;
  a2.prev = prev_score;
  a2.off = sent_offsets;
  a2.tok = out_token;
  a2.par = out_parent;
  a2.score = out_score;
  a2.row_lse = out_row_lse;
  hipError_t e = kb::launch_k2(a2, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(KB_ERR_HIP, "merge kernel launch: %s", hipGetErrorString(e));
  return ok();
}

kb_status kb_standin_alive(int S, const int32_t* S_dev, int k, int t, const int32_t* sid, const int32_t* lengths,
                     uint8_t* alive, void* stream) {
  if (S < 0 || k < 1) return fail(KB_ERR_INVALID_ARG, "S = %d, k = %d", S, k);
  if ((long long)S * k > INT_MAX) return fail(KB_ERR_UNSUPPORTED, "S*k does not fit in int32");
  if (S == 0) return ok();
  if (!sid || !lengths || !alive) return fail(KB_ERR_INVALID_ARG, "null sid, lengths or alive");
  hipError_t e = kb::launch_standin_alive(S, S_dev, k, t, sid, lengths, alive,
                                          reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(KB_ERR_HIP, "stand-in alive kernel launch: %s", hipGetErrorString(e));
  return ok();
}

kb_status kb_standin_step(int S, const int32_t* S_dev, int k, int t, const int32_t* sid, const int32_t* lengths,
                          const float* score, int32_t* keep_idx, int32_t* counts, int32_t* new_sent_offsets,
                          float* prev_next, int32_t* sid_next, uint8_t* alive, int32_t* counts_host,
                          const void* table, int T, void* next_h, size_t row_bytes, void* stream) {
  if (S < 0 || k < 1) return fail(KB_ERR_INVALID_ARG, "S = %d, k = %d", S, k);
  if ((long long)S * k > INT_MAX) return fail(KB_ERR_UNSUPPORTED, "S*k does not fit in int32");
  if (k >= (1 << 10)) return fail(KB_ERR_UNSUPPORTED, "k = %d: at most 1023 entries per sentence", k);
  if (!counts || !new_sent_offsets) return fail(KB_ERR_INVALID_ARG, "null counts or new_sent_offsets");
  if (S > 0 && (!sid || !lengths || !score || !keep_idx || !prev_next || !sid_next))
    return fail(KB_ERR_INVALID_ARG, "null sid, lengths, score, keep_idx, prev_next or sid_next");
  if (next_h) {
    if (!table) return fail(KB_ERR_INVALID_ARG, "null table with next_h");
    if (t < 0 || T < 1 || t + 1 >= T) return fail(KB_ERR_INVALID_ARG, "t = %d, T = %d: next states need t + 1 < T", t, T);
    if (row_bytes == 0 || row_bytes % 4 != 0)
      return fail(KB_ERR_INVALID_ARG, "row_bytes must be a positive multiple of 4");
    if (row_bytes / 4 > INT_MAX) return fail(KB_ERR_UNSUPPORTED, "row too long");
    if (!aligned(table, 4) || !aligned(next_h, 4))
      return fail(KB_ERR_INVALID_ARG, "table and next_h must be 4-byte aligned");
  }
  hipError_t e = kb::launch_standin_step(S, S_dev, k, t, sid, lengths, score, keep_idx, counts, new_sent_offsets,
                                         prev_next, sid_next, alive, counts_host, table, T, next_h, row_bytes,
                                         reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(KB_ERR_HIP, "stand-in step kernel launch: %s", hipGetErrorString(e));
  return ok();
}

kb_status kb_standin_next_h(int n_max, const int32_t* n_dev, int k, int T, int t, const int32_t* keep, const int32_t* sid,
                      const void* table, void* out, size_t row_bytes, void* stream) {
  if (n_max < 0 || k < 1 || T < 1 || t < 0 || t >= T)
    return fail(KB_ERR_INVALID_ARG, "n_max = %d, k = %d, T = %d, t = %d", n_max, k, T, t);
  if (row_bytes == 0 || row_bytes % 4 != 0) return fail(KB_ERR_INVALID_ARG, "row_bytes must be a positive multiple of 4");
  if (row_bytes / 4 > INT_MAX) return fail(KB_ERR_UNSUPPORTED, "row too long");
  if (n_max == 0) return ok();
  if (!keep || !sid || !table || !out) return fail(KB_ERR_INVALID_ARG, "null keep, sid, table or out");
  if (!aligned(table, 4) || !aligned(out, 4)) return fail(KB_ERR_INVALID_ARG, "table and out must be 4-byte aligned");
  hipError_t e = kb::launch_standin_next_h(n_max, n_dev, k, T, t, keep, sid, table, out, row_bytes,
                                           reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(KB_ERR_HIP, "stand-in state gather launch: %s", hipGetErrorString(e));
  return ok();
}

}  // extern "C"
