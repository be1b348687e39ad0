// K1, wide variant: the fused output-layer projection for many live rows
// (bf16 h and W, H % 128 == 0, V % 8 == 0, 16-byte aligned operands).
//
// Tile: 256 words x 256 hypothesis rows per workgroup of four waves; wave
// (wv, wh) owns words [128 wv, 128 wv + 128) and rows [128 wh, 128 wh + 128)
// as 4 x 4 accumulators of v_mfma_f32_32x32x16_bf16 (256 registers, kept in
// the accumulation registers).  A square tile moves 1 KB of operands per 16
// states for 131k flops, half the operand bytes per flop of a 128 x 256 tile,
// which keeps the global->LDS stream well below what a CU can sustain.
//
// Operands reach LDS through a ring of four stages (32 states each) filled by
// the gfx950 global->LDS DMA, with a wave-uniform base in SGPRs and fixed
// per-lane offsets, so issuing a stage costs eight instructions per wave.
// Layouts and swizzles are those of the narrow DMA kernel: W stays
// V-contiguous (A-fragments via the LDS transpose read), h rows are
// row-major 64-byte slices per stage.
//
// Per stage the wave runs the first half's 16 MFMAs while it reads the
// second half's fragments and issues the W rows of the stage three ahead
// (into the buffer every wave finished before the previous barrier), waits
// for the next stage and passes the only barrier of the stage, then runs the
// second half's MFMAs while it reads the next stage's first fragments and
// issues the h rows of the stage three ahead.  LDS reads and DMA issue
// therefore always overlap MFMAs, and no wait drains the ring.
//
// Epilogue per tile (the accumulators start at the bias, so Algorithm 3's
// AddBias costs nothing; words >= V start at -inf and drop out everywhere):
//   * per row of the lane: tile max (3-input max tree), then the running
//     (max, sum) with one rescale per tile (Algorithm 4's identity);
//   * rows whose tile max reaches max(local k-th best, shared threshold)
//     append their candidates to a per-row LDS list; the owner thread of the
//     row inserts them into its sorted k-list (registers) and raises the
//     thresholds.  Ties are kept by the filter and settled by word index.
#pragma once

#include <type_traits>

#include "k1_common.hpp"

namespace kb {

__device__ __forceinline__ float fmax3(float a, float b, float c) { return fmaxf(fmaxf(a, b), c); }

struct WideGeom {
  static constexpr int BV = 256, BH = 256, BK = 32;
  static constexpr int WE = BK * BV;  // bf16 elements of W per stage
  static constexpr int HE = BH * BK;  // bf16 elements of h per stage
  static constexpr int OPS = 8;       // DMA instructions per wave per stage
  static constexpr int DMA_SLOT0 = 8; // first MFMA (of each 16) followed by a DMA instruction
  static constexpr int CAPH = 8;      // candidate slots per row and holder per round
  static constexpr int DONE = 64;     // "no pending candidates" position
  static constexpr int MS = 16;       // splits that share their running row maxima
};

struct alignas(16) WideEpi {
  float bias[2][WideGeom::BV];    // bias of the current / next tile (DMA)
  uint32_t tgk[2][WideGeom::BH];  // shared-threshold keys read for the current / next tile (DMA)
  float thr[WideGeom::BH];        // row's local threshold: its k-th best so far, or the seed
  uint32_t cnt[WideGeom::BH];     // candidates each holder appended to the row this round (one byte each)
  int flag[4];                    // "a lane could not append" of this and the next round
  float trash_x[4 * 64];          // per lane: where a score that takes no slot is written
  uint8_t trash_p[4 * 64];
  union {
    // positions (0..63), among the holder's scores, of the scores appended this
    // round per row and holder; the scores themselves go to the idle ring buffer
    uint8_t p[WideGeom::BH][4][WideGeom::CAPH];
    float red[WideGeom::BH][16];  // seeds, then the per-holder statistics
  } u;
};

// Candidate scores of a round live in the ring buffer of a tile's last stage
// (nk is a multiple of 4, so that is always buffer 3): its reads end at the
// barrier in the middle of that stage, and the next DMA into it is issued in
// the next tile's first stage, after the epilogue's last barrier.  Slot c of
// (row r, holder h) is float (4 r + h) * CAPH + (c ^ ((r >> 1) & 7)): the XOR
// spreads a wave's appends (32 rows x 2 holders, any slot) over 32 banks.
__device__ __forceinline__ int cand_slot(int r, int h, int c) {
  return (r * 4 + h) * WideGeom::CAPH + (c ^ ((r >> 1) & 7));
}
static_assert(WideGeom::CAPH == 8, "the slot swizzle permutes 8 slots");
static_assert(WideGeom::BH * 4 * WideGeom::CAPH * 4 <= (WideGeom::WE + WideGeom::HE) * 2,
              "a round's candidate scores fit in one ring buffer");

// Global->LDS DMA with a wave-uniform base (SGPR pair) and a per-lane 32-bit
// byte offset: lane i copies 16 bytes from base + voff + OFF to LDS byte
// M0 + OFF + 16 i (the immediate offset shifts both addresses).
// Group form: M0 is set once (set_m0) for up to four DMA instructions whose
// immediate offsets (0..3072) shift both the global and the LDS address; the
// per-lane offset is pre-compensated by -OFF.
__device__ __forceinline__ void set_m0(uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0" ::"s"(__builtin_amdgcn_readfirstlane(lds_base)) : "m0");
}
// A vector memory instruction that reads an SGPR needs 5 wait states after a
// VALU instruction that wrote it (v_readfirstlane, or the v_readlane that
// restores a spilled SGPR); the compiler inserts them for its own
// instructions, not for inline assembly.  The build checks the device
// assembly of this file for the hazard on every path (isa_check.py).  Here,
// in the main loop, the base pair is a loop invariant that the compiler keeps
// in SGPRs; load4_async below guards itself.
template <int OFF>
__device__ __forceinline__ void dma16_off(uint32_t voff, const void* sbase) {
  const uint64_t p = reinterpret_cast<uint64_t>(sbase);
  const uint64_t u = ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(p >> 32)) << 32) |
                     (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)p);
  asm volatile("global_load_lds_dwordx4 %0, %1 offset:%2" ::"v"(voff), "s"(reinterpret_cast<const void*>(u)), "i"(OFF));
}

// Marks an accumulator block as redefined in place (it stays in the
// accumulation registers).  Used at the start of each row's epilogue work so
// that the compiler copies only that row's 64 scores into VGPRs, and copies
// them again in each candidate round instead of keeping all 256 alive.
__device__ __forceinline__ void opaque(f32x16& x) { asm volatile("" : "+a"(x)); }

// A row's results "used" at a point that, being volatile, stays ordered
// before the next row's opaque(): together they keep the compiler from
// interleaving consecutive rows (which would hold several rows' 64 scores in
// VGPRs at once).
__device__ __forceinline__ void done(float x) { asm volatile("" ::"v"(x)); }
__device__ __forceinline__ void done(int x) { asm volatile("" ::"v"(x)); }

// 64-bit order key of a (score, word) candidate: higher score first, then
// lower word (the strict-'>' scans of the paper).  -0 is folded into +0 so
// that equal scores compare equal.
__device__ __forceinline__ uint64_t cand_key(float x, int word) {
  return ((uint64_t)f2key(x + 0.0f) << 32) | (uint32_t)~(uint32_t)word;
}

// Global atomic max and 16-byte load issued from inline assembly: the
// compiler then adds no waits of its own for them (its conservative
// vmcnt(0) would also wait for the DMA stages in flight).  The atomic's
// completion is never waited for; the load is waited for with load_wait.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void atomic_umax_nowait(uint32_t* p, uint32_t v) {
  asm volatile("global_atomic_umax %0, %1, off" ::"v"(p), "v"(v) : "memory");
}
// 4-byte load from a wave-uniform base (SGPR pair) plus a per-lane byte offset.
// The base is first copied by a scalar move into a pair of the statement's
// own (a scalar instruction waits for a VALU write by itself, and a scalar
// write needs no wait states before the load): the loads run in the
// epilogue, where register pressure can make the compiler spill the base
// pair and restore it with v_readlane right before them (unguarded, builds
// that did so read a stale base and faulted).
__device__ __forceinline__ uint32_t load4_async(uint32_t voff, const void* sbase) {
  const uint64_t p = reinterpret_cast<uint64_t>(sbase);
  const uint64_t u = ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(p >> 32)) << 32) |
                     (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)p);
  uint32_t v;
  uint64_t t;
  asm volatile("s_mov_b64 %1, %3\n\tglobal_load_dword %0, %2, %1" : "=v"(v), "=&s"(t) : "v"(voff), "s"(u));
  return v;
}
// every vector memory operation of the wave done; the registers pass
// through so that their uses stay behind the wait
__device__ __forceinline__ void load_wait(uint32_t (&v)[16]) {
  asm volatile("s_waitcnt vmcnt(0)"
               : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]), "+v"(v[4]), "+v"(v[5]), "+v"(v[6]), "+v"(v[7]),
                 "+v"(v[8]), "+v"(v[9]), "+v"(v[10]), "+v"(v[11]), "+v"(v[12]), "+v"(v[13]), "+v"(v[14]),
                 "+v"(v[15]));
}

__device__ __forceinline__ float max4(const f32x16& x, int q) {
  return fmaxf(fmax3(x[4 * q], x[4 * q + 1], x[4 * q + 2]), x[4 * q + 3]);
}

// What the kernel does with its tiles of scores.
enum WideMode {
  kWideKBest = 0,   // bias, softmax statistics, per-split k-best (the fused step)
  kWideArgmax = 1,  // the greedy (beam 1) form of Algorithm 5: only the best word of
                    // every row, no softmax statistics (nothing written to a.stats)
  kWideStore = 2,   // the plain projection p = W h: every score stored to a.logits
                    // (N x V float32, row-major), nothing else (the unfused baseline)
};

template <int KC, int MODE = kWideKBest>
__global__ __launch_bounds__(256, 1) void k1_wide(K1Args a) {
  constexpr bool STATS = MODE == kWideKBest;
  using G = WideGeom;
  constexpr int BV = G::BV, BH = G::BH, BK = G::BK, WE = G::WE, HE = G::HE;
  __shared__ __attribute__((aligned(16))) uint16_t S0[WE + HE], S1[WE + HE], S2[WE + HE], S3[WE + HE];
  __shared__ WideEpi ep;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wv = wave & 1, wh = wave >> 1;
  const int half = lane >> 5, col = lane & 31;
  const int holder = wv * 2 + half;  // which of the row's four holders this lane is
  const int k = a.k;

  int row_tile, split;
  k1_cell(a, blockIdx.x, row_tile, split);
  const int h0 = row_tile * BH;
  // the split's tiles are split, split + P, split + 2P, ...: interleaved, so
  // every split meets the high-scoring words of a skewed bias (low word ids
  // under a Zipf-like prior) early and no split is left with all of them
  const int nt = (a.n_vtiles - split + a.P - 1) / a.P;
  const int nk = a.H / BK;  // a multiple of 4: every tile starts on ring buffer 0
  const int total = nt * nk;

  // ---- per-lane DMA byte offsets (fixed for the whole kernel)
  // W slot s = 256 wave + 64 i + lane: stage row r = s / 32, physical chunk
  // s % 32 holding logical chunk (s % 32) ^ wswz(r).
  // h slot s: row n = s / 4, physical chunk s % 4 holding chunk (s % 4) ^ hswz(n).
  // Offsets are pre-compensated for the immediate offset 1024 i of DMA
  // instruction i (they stay >= 0: r >= 2 i and V >= 256; n >= 16 i and H >= 128).
  uint32_t woff[4], hoff[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = wave * 8 + i * 2 + half;
    woff[i] = (uint32_t)r * (uint32_t)a.V * 2u + (uint32_t)((col ^ wswz(r)) * 16) - 1024u * i;
    const int n = wave * 64 + i * 16 + (lane >> 2);
    hoff[i] = (uint32_t)min(h0 + n, a.N - 1) * (uint32_t)a.H * 2u + (uint32_t)(((lane & 3) ^ hswz(n)) * 16) - 1024u * i;
  }

  // ---- the next stage to issue: tile start iv0 (tile it), state offset ik0;
  // wsrc / hsrc point at its first W row / h column; wdma are the W offsets of
  // its tile (clamped for the last, ragged tile: words >= V read word V - 8..
  // instead, which start at -inf).
  int iv0 = split * BV, ik0 = 0, it = 0, issued = 0;
  const char* wsrc = reinterpret_cast<const char*>(a.W) + (size_t)iv0 * 2;
  const char* hsrc = reinterpret_cast<const char*>(a.h);
  uint32_t wdma[4];
  auto set_wdma = [&]() {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      wdma[i] = woff[i];
      if (iv0 + BV > a.V) {
        const int r = wave * 8 + i * 2 + half;
        wdma[i] = (uint32_t)r * (uint32_t)a.V * 2u + (uint32_t)(min(iv0 + (col ^ wswz(r)) * 8, a.V - 8) - iv0) * 2u -
                  1024u * i;
      }
    }
  };
  set_wdma();
  // DMA instruction i (0..7) of the next stage into buffer buf: W rows (i < 4)
  // or h rows; i = 0 and 4 set M0 for their group of four
  auto dma_part = [&](uint16_t* buf, int i) {
    const uint32_t sb = lds_addr(buf) + wave * 4096 + (i < 4 ? 0 : WE * 2);
    if ((i & 3) == 0) set_m0(sb);
    switch (i) {
      case 0: dma16_off<0>(wdma[0], wsrc); break;
      case 1: dma16_off<1024>(wdma[1], wsrc); break;
      case 2: dma16_off<2048>(wdma[2], wsrc); break;
      case 3: dma16_off<3072>(wdma[3], wsrc); break;
      case 4: dma16_off<0>(hoff[0], hsrc); break;
      case 5: dma16_off<1024>(hoff[1], hsrc); break;
      case 6: dma16_off<2048>(hoff[2], hsrc); break;
      default: dma16_off<3072>(hoff[3], hsrc); break;
    }
  };
  auto dma_finish = [&]() {  // the tile's bias rides with its first stage
    if (ik0 == 0 && wave == 0) dma16(a.b + min(iv0 + lane * 4, a.V - 4), lds_addr(&ep.bias[it & 1][0]));
    ++issued;
    ik0 += BK;
    wsrc += (size_t)BK * a.V * 2;
    hsrc += BK * 2;
    if (ik0 == a.H) {
      ik0 = 0;
      iv0 += a.P * BV;
      ++it;
      wsrc = reinterpret_cast<const char*>(a.W) + (size_t)iv0 * 2;
      hsrc = reinterpret_cast<const char*>(a.h);
      set_wdma();
    }
  };
  auto issue_whole = [&](uint16_t* buf) {
    if (issued < total) {
#pragma unroll
      for (int i = 0; i < G::OPS; ++i) dma_part(buf, i);
      dma_finish();
    }
  };

  // ---- MFMA fragments of one 16-state step (kk) of a stage.  Per-lane byte
  // offsets within a stage buffer: A (W^T) fragments of block vb at kk = 0
  // (kk adds 16 rows, which leaves the swizzle unchanged); B (h) fragments of
  // block 0 at each kk (blocks are 32 rows = 2 KB apart, same swizzle).
  uint32_t aoff[4], boff[2];
  {
    const int g = lane >> 4, j = lane & 15;
    const int r0 = 8 * (g >> 1) + (j >> 2);
#pragma unroll
    for (int vb = 0; vb < 4; ++vb) {
      const int colw = wv * 128 + vb * 32 + 16 * (g & 1) + 4 * (j & 3);
      aoff[vb] = (uint32_t)(r0 * BV + (((colw >> 3) ^ wswz(r0)) << 3) + (colw & 7)) * 2u;
    }
    const int n = wh * 128 + col;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) boff[kk] = (uint32_t)(WE + n * 32 + (((kk * 2 + half) ^ hswz(n)) * 8)) * 2u;
  }
  // A fragment of block vb = two transpose reads (states 0-3 and 4-7 of the
  // lane's half); B fragment of block hb = one 16-byte read.
  struct Frag {
    s16x4 lo[4], hi[4];
    bf16x8 b[4];
  };
  // read u (0..11) of a fragment set, in the order the MFMAs consume them:
  // b0, lo0, hi0, b1, b2, b3, lo1, hi1, lo2, hi2, lo3, hi3
  auto rd = [&](const uint16_t* buf, int kk, int u, Frag& f) {
    const KB_LDS char* base = (const KB_LDS char*)(const KB_LDS void*)buf;
    constexpr int kind[12] = {2, 0, 1, 2, 2, 2, 0, 1, 0, 1, 0, 1};  // 0 lo, 1 hi, 2 b
    constexpr int blk[12] = {0, 0, 0, 1, 2, 3, 1, 1, 2, 2, 3, 3};
    const int x = blk[u];
    if (kind[u] == 2) {
      f.b[x] = *(const KB_LDS bf16x8*)(base + boff[kk] + x * 2048);
    } else {
      const KB_LDS char* p = base + aoff[x] + kk * 16 * BV * 2 + kind[u] * 4 * BV * 2;
      const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((KB_LDS s16x4*)p);
      if (kind[u] == 0)
        f.lo[x] = v;
      else
        f.hi[x] = v;
    }
  };

  f32x16 acc[4][4];
  auto mf = [&](const Frag& f, int i) {  // MFMA i of a 16-state step: block (i / 4, i % 4)
    const int vb = i >> 2, hb = i & 3;
    const bf16x8 fa = __builtin_bit_cast(bf16x8, __builtin_shufflevector(f.lo[vb], f.hi[vb], 0, 1, 2, 3, 4, 5, 6, 7));
    acc[vb][hb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa, f.b[hb], acc[vb][hb], 0, 0, 0);
  };

  // ---- accumulators start at the tile's bias; words >= V at -inf
  auto init_acc = [&](int ti) {  // ti: the tile's ordinal within the split
    const int par = ti & 1;
    const int v0 = (split + ti * a.P) * BV;
    const bool ragged = v0 + BV > a.V;
    // word of (vb, i, j) is valid iff vb * 32 + 8 i + j < lim
    const int lim = a.V - v0 - wv * 128 - 4 * half;
#pragma unroll
    for (int vb = 0; vb < 4; ++vb) {
      f32x16 bv;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int wl = wv * 128 + vb * 32 + 8 * i + 4 * half;
        float4 bb = *reinterpret_cast<const float4*>(&ep.bias[par][wl]);
        if constexpr (MODE == kWideStore) bb = make_float4(0.f, 0.f, 0.f, 0.f);  // p = W h only
        bv[4 * i + 0] = bb.x;
        bv[4 * i + 1] = bb.y;
        bv[4 * i + 2] = bb.z;
        bv[4 * i + 3] = bb.w;
        if (ragged) {
#pragma unroll
          for (int j = 0; j < 4; ++j)
            if (vb * 32 + 8 * i + j >= lim) bv[4 * i + j] = -INFINITY;
        }
      }
#pragma unroll
      for (int hb = 0; hb < 4; ++hb) {
        acc[vb][hb] = bv;
        opaque(acc[vb][hb]);  // written straight into the accumulation registers
      }
    }
  };

  // ---- epilogue state
  float st_m[4], st_s[4];  // running (max, sum of exp(x - max)) of the lane's rows
  // owner (row = tid): the k best (score, word) of the split so far as
  // descending 64-bit keys; the first KC - k slots hold sentinels above any key
  uint64_t lkey[KC];
  float published = kNoThr;
  float rowbest = kNoThr, shared_best = kNoThr;  // best listed score of the row, and the one shared
#pragma unroll
  for (int hb = 0; hb < 4; ++hb) {
    st_m[hb] = kStatInit;
    st_s[hb] = 0.f;
  }
#pragma unroll
  for (int j = 0; j < KC; ++j) lkey[j] = (j < KC - k) ? ~0ull : 0ull;
  ep.thr[tid] = kNoThr;
  ep.cnt[tid] = 0u;
  if (tid < 4) ep.flag[tid] = 0;

  auto publish = [&](float v) {
    if (h0 + tid < a.N && v > published) {
      atomic_umax_nowait(&a.gthr[h0 + tid], f2key(v));
      published = v;
    }
  };

  // splits 0..MS-1 share their best row scores (k > 12: the longer k-list
  // leaves no registers for the maxima; not used)
  constexpr bool kShare = KC <= 12;
  auto epilogue = [&](int ti) {
    const int par = ti & 1;
    const int v0 = (split + ti * a.P) * BV;
    // the running maxima splits 0..MS-1 have shared for the owner's row
    // (loaded now, used after the statistics; split-major, so each load of
    // the wave reads 64 consecutive rows)
    uint32_t key[G::MS];
    if (kShare && ti > 0) {
      const size_t stride = (size_t)a.row_tiles * BH;
#pragma unroll
      for (int i = 0; i < G::MS; ++i) key[i] = load4_async(4u * tid, a.gmax + h0 + i * stride);
    }
    float tmax[4];
    // statistics (Algorithm 4, one rescale per tile)
#pragma unroll
    for (int hb = 0; hb < 4; ++hb) {
#pragma unroll
      for (int vb = 0; vb < 4; ++vb) opaque(acc[vb][hb]);
      float m0 = fmax3(acc[0][hb][0], acc[0][hb][1], acc[0][hb][2]);
      float m1 = fmax3(acc[0][hb][3], acc[0][hb][4], acc[0][hb][5]);
#pragma unroll
      for (int vb = 0; vb < 4; ++vb)
#pragma unroll
        for (int r = (vb == 0 ? 6 : 0); r < 16; r += 4) {
          m0 = fmax3(m0, acc[vb][hb][r], acc[vb][hb][r + 1]);
          m1 = fmax3(m1, acc[vb][hb][r + 2], acc[vb][hb][r + 3]);
        }
      const float mx = fmaxf(m0, m1);
      tmax[hb] = mx;
      if constexpr (!STATS) {
        done(mx);
        continue;
      }
      const float mnew = fmaxf(st_m[hb], mx);
      const float ml2 = mnew * kL2E;
      float s0 = st_s[hb] * exp2_fast((st_m[hb] - mnew) * kL2E), s1 = 0.f;
#pragma unroll
      for (int vb = 0; vb < 4; ++vb)
#pragma unroll
        for (int r = 0; r < 16; r += 2) {
          s0 += exp2_fast(fmaf(acc[vb][hb][r], kL2E, -ml2));
          s1 += exp2_fast(fmaf(acc[vb][hb][r + 1], kL2E, -ml2));
        }
      st_s[hb] = s0 + s1;
      st_m[hb] = mnew;
      done(st_s[hb]);
      done(mx);
    }
    if (kShare && ti > 0) {
      // the k-th largest of the shared maxima: they are scores of k distinct
      // words of the row, so it is a lower bound of the row's k-th best.  It
      // is worked out only where at least k of them beat the row's present
      // threshold (else it cannot raise it): insertion into a right-aligned
      // descending list by median-of-three.
      load_wait(key);  // long landed: issued before the statistics
      const uint32_t tk = max(f2key(ep.thr[tid]), ep.tgk[par][tid]);
      int above = 0;
#pragma unroll
      for (int i = 0; i < G::MS; ++i) above += key[i] > tk ? 1 : 0;
      if (__builtin_amdgcn_ballot_w64(above >= k) != 0ull) {
        float kv[KC];
#pragma unroll
        for (int j = 0; j < KC; ++j) kv[j] = (j < KC - k) ? INFINITY : -INFINITY;
#pragma unroll
        for (int i = 0; i < G::MS; ++i) {
          const float x = key2f(key[i]);
#pragma unroll
          for (int j = KC - 1; j > 0; --j) kv[j] = __builtin_amdgcn_fmed3f(kv[j - 1], kv[j], x);
          kv[0] = fmaxf(kv[0], x);
        }
        const float t2 = kv[KC - 1];
        if (above >= k && t2 > ep.thr[tid]) {
          ep.thr[tid] = t2;
        }
      }
      lds_barrier();  // the holders read the raised threshold below
    }

    // first tile of the split: seed each row's threshold.  Every holder finds
    // the 4 largest of its 16 quad maxima; these 16 distinct scores of the row
    // are gathered and their k-th largest (k <= 16) is a valid threshold: k
    // scores of the row are >= it.
    if (ti == 0) {
#pragma unroll
      for (int hb = 0; hb < 4; ++hb) {
#pragma unroll
        for (int vb = 0; vb < 4; ++vb) opaque(acc[vb][hb]);
        float sv[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
#pragma unroll
        for (int vb = 0; vb < 4; ++vb)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            float x = max4(acc[vb][hb], q);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const float hi = fmaxf(sv[j], x);
              x = fminf(sv[j], x);
              sv[j] = hi;
            }
          }
        *reinterpret_cast<float4*>(&ep.u.red[wh * 128 + hb * 32 + col][4 * holder]) =
            make_float4(sv[0], sv[1], sv[2], sv[3]);
        done(sv[3]);
      }
      lds_barrier();
      {
        // k-th largest of the 16: right-aligned list of KC slots, +inf sentinels first
        float kv[KC];
#pragma unroll
        for (int j = 0; j < KC; ++j) kv[j] = (j < KC - k) ? INFINITY : -INFINITY;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          float x = ep.u.red[tid][i];
#pragma unroll
          for (int j = 0; j < KC; ++j) {
            const float hi = fmaxf(kv[j], x);
            x = fminf(kv[j], x);
            kv[j] = hi;
          }
        }
        const float seed = kv[KC - 1];
        if (seed > ep.thr[tid]) {
          ep.thr[tid] = seed;
        }
      }
      lds_barrier();
    }

    // candidate rounds.  A lane appends, in position order, every score >= the
    // row's threshold to its own CAPH slots of the row; past CAPH it notes the
    // first position it could not append and resumes there in the next round,
    // against the raised threshold.  Quads are skipped unless some lane of the
    // wave needs them; inside a quad every lane stores each score, to its next
    // slot or to its own discard slot, so the appends take no branch.
    int resume[4];
#pragma unroll
    for (int hb = 0; hb < 4; ++hb) {
      const int rl = wh * 128 + hb * 32 + col;
      const float t = fmaxf(ep.thr[rl], key2f(ep.tgk[par][rl]));
      resume[hb] = tmax[hb] >= t ? 0 : G::DONE;
    }
    for (int round = 0;; ++round) {
      int ovf = 0;
#pragma unroll
      for (int hb = 0; hb < 4; ++hb) {
        const int rs = resume[hb];
        if (__builtin_amdgcn_ballot_w64(rs < G::DONE) != 0ull) {
          const int rl = wh * 128 + hb * 32 + col;
          // lanes with nothing pending on this row compare against +inf
          const float t = rs < G::DONE ? fmaxf(ep.thr[rl], key2f(ep.tgk[par][rl])) : INFINITY;
          int newres = G::DONE, c = 0;
          // the lane's slots of the row (LDS byte addresses, opaque so that the
          // per-slot addresses are formed at the store, not kept in registers)
          uint32_t sx = lds_addr(S3) + 4u * (uint32_t)((rl * 4 + holder) * G::CAPH), sp = lds_addr(&ep.u.p[rl][holder][0]);
          const int swz = (rl >> 1) & 7;
          uint32_t tx = lds_addr(&ep.trash_x[tid]), tp = lds_addr(&ep.trash_p[tid]);
          asm volatile("" : "+v"(sx), "+v"(sp), "+v"(tx), "+v"(tp));
#pragma unroll
          for (int vb = 0; vb < 4; ++vb) {
            opaque(acc[vb][hb]);  // only this block's 16 scores in VGPRs at a time
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const bool qp = max4(acc[vb][hb], q) >= t && vb * 16 + 4 * q + 3 >= rs;
              if (__builtin_amdgcn_ballot_w64(qp) != 0ull) {  // a uniform skip for most quads
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                  const int pos = vb * 16 + 4 * q + j;
                  const float x = acc[vb][hb][4 * q + j];
                  const bool pred = x >= t && pos >= rs;
                  const bool room = c < G::CAPH;
                  newres = (pred && !room) ? min(newres, pos) : newres;
                  const bool ok = pred && room;
                  int pv = pos;  // materialized here, not hoisted (64 constants would pin VGPRs)
                  asm volatile("" : "+v"(pv));
                  // every lane stores: a score that takes no slot goes to the lane's own
                  // discard slot, so the appends need no branch
                  *(KB_LDS float*)(uintptr_t)(ok ? sx + 4 * (c ^ swz) : tx) = x;
                  *(KB_LDS uint8_t*)(uintptr_t)(ok ? sp + c : tp) = (uint8_t)pv;
                  c += ok ? 1 : 0;
                }
              }
            }
            done(c);
          }
          reinterpret_cast<uint8_t*>(&ep.cnt[rl])[holder] = (uint8_t)c;
          resume[hb] = newres;
          ovf |= newres != G::DONE;
          done(newres);
        }
      }
      if (ovf) ep.flag[round & 1] = 1;
      lds_barrier();
      if (tid == 0) ep.flag[(round + 1) & 1] = 0;  // read only after the next barrier
      {
        const uint32_t cw = ep.cnt[tid];
        if (cw != 0u) {
          // the row's candidates, holder after holder, as one sequence: the
          // wave loops as long as its longest row, not its longest holder of
          // each holder in turn
          const int c0 = cw & 0xFF, c1 = (cw >> 8) & 0xFF, c2 = (cw >> 16) & 0xFF;
          const int e1 = c0, e2 = c0 + c1, e3 = e2 + c2, tot = e3 + (int)(cw >> 24);
          for (int i = 0; i < tot; ++i) {
            const int hd = (i >= e1 ? 1 : 0) + (i >= e2 ? 1 : 0) + (i >= e3 ? 1 : 0);
            const int j = i - (hd == 0 ? 0 : (hd == 1 ? e1 : (hd == 2 ? e2 : e3)));
            const int p = ep.u.p[tid][hd][j];
            const float cx = *(KB_LDS const float*)(uintptr_t)(lds_addr(S3) + 4u * (uint32_t)cand_slot(tid, hd, j));
            // word of position p of holder hd: holder = 2 wv + half
            const int word = v0 + (hd >> 1) * 128 + (hd & 1) * 4 + (p >> 4) * 32 + ((p >> 2) & 3) * 8 + (p & 3);
            uint64_t key = cand_key(cx, word);
            {
              rowbest = key > lkey[KC - 1] ? fmaxf(rowbest, cx) : rowbest;
              // insertion with independent compares, without a branch: the keys
              // are descending, so gt[] is false then true and the key lands at
              // the first true; a key below the k-th leaves gt[] all false and
              // the list unchanged
              bool gt[KC];
#pragma unroll
              for (int jj = 0; jj < KC; ++jj) gt[jj] = key > lkey[jj];
#pragma unroll
              for (int jj = KC - 1; jj > 0; --jj) lkey[jj] = gt[jj] ? (gt[jj - 1] ? lkey[jj - 1] : key) : lkey[jj];
              lkey[0] = gt[0] ? key : lkey[0];
            }
          }
          ep.cnt[tid] = 0u;
        }
        const float kth = key2f((uint32_t)(lkey[KC - 1] >> 32));
        if (kth > ep.thr[tid]) ep.thr[tid] = kth;
      }
      lds_barrier();
      if (ep.flag[round & 1] == 0) break;
    }
    // shared on the split's tiles 0, 1, 2, 4, 8, ... only (device-wide
    // atomics are written through to memory; a stale value is still a valid
    // bound): the row's threshold, and the best score of the row this split
    // has listed (its maximum, unless that never reached a threshold; any
    // score of the split is a valid entry of the shared maxima)
    if ((ti & (ti - 1)) == 0) publish(ep.thr[tid]);
    if (kShare && split < G::MS && (ti & (ti - 1)) == 0 && rowbest > shared_best && h0 + tid < a.N) {
      atomic_umax_nowait(&a.gmax[(size_t)split * a.row_tiles * BH + h0 + tid], f2key(rowbest));
      shared_best = rowbest;
    }
  };

  // ---- the plain projection: the tile's scores to a.logits (rows < N,
  // words < V; each lane holds 4 consecutive words of a row per 16-byte store)
  auto store_tile = [&](int ti) {
    const int v0 = (split + ti * a.P) * BV;
#pragma unroll
    for (int hb = 0; hb < 4; ++hb) {
      const int n = h0 + wh * 128 + hb * 32 + col;
#pragma unroll
      for (int vb = 0; vb < 4; ++vb) {
        opaque(acc[vb][hb]);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int w = v0 + wv * 128 + vb * 32 + 8 * i + 4 * half;
          if (n < a.N && w < a.V)
            *reinterpret_cast<float4*>(a.logits + (size_t)n * a.V + w) =
                make_float4(acc[vb][hb][4 * i], acc[vb][hb][4 * i + 1], acc[vb][hb][4 * i + 2], acc[vb][hb][4 * i + 3]);
        }
      }
    }
  };

  // ---- the stage pipeline
  uint16_t* const bufs[4] = {S0, S1, S2, S3};
  Frag F0, F1;

  // three stages ahead: stage g + 3 goes into the buffer of stage g - 1,
  // which every wave finished reading before the barrier of stage g - 1
  issue_whole(S0);
  issue_whole(S1);
  issue_whole(S2);
  // stage 0 landed: at most the two later stages outstanding
  if (total >= 3)
    wait_vm<2 * G::OPS>();
  else if (total == 2)
    wait_vm<G::OPS>();
  else
    wait_vm<0>();
  lds_barrier();
  init_acc(0);
#pragma unroll
  for (int u = 0; u < 12; ++u) rd(S0, 0, u, F0);

  // One stage (32 states) on buffer b.  LDS reads (two per MFMA, early, so
  // they have landed before their use) and DMA instructions (one per MFMA,
  // spread over the whole stage so the address unit is never flooded) sit
  // between MFMAs, where their issue hides behind the MFMA pipe:
  //   16 MFMAs on F0 (first 16 states), reading F1 (second 16) and issuing
  //   the W rows of stage g + 3 into buffer b - 1;
  //   wait for stage g + 1, barrier;
  //   16 MFMAs on F1, reading F0 of stage g + 1 and issuing the h rows of
  //   stage g + 3.
  int g = 0;
  auto body = [&](auto bc, auto rc) {
    constexpr int b = decltype(bc)::value;
    constexpr bool read_next = decltype(rc)::value;  // false in a tile's last stage: the next
                                                     // tile's first fragments are read after
                                                     // the epilogue (keeps VGPRs free for it)
    uint16_t* const cur = bufs[b];
    uint16_t* const nxt = bufs[(b + 1) & 3];
    uint16_t* const fill = bufs[(b + 3) & 3];
    const bool more = issued < total;  // stage g + 3 exists
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      mf(F0, i);
      if (i < 6) {
        rd(cur, 1, 2 * i, F1);
        rd(cur, 1, 2 * i + 1, F1);
      }
      if (more && i >= G::DMA_SLOT0 && i < G::DMA_SLOT0 + 4) dma_part(fill, i - G::DMA_SLOT0);
      __builtin_amdgcn_sched_barrier(0);
    }
    if (g + 1 < total) {
      // DMA instructions issued after stage g + 1's: stage g + 2 (whole) and
      // the W half of stage g + 3
      if (g + 3 < total)
        wait_vm<G::OPS + G::OPS / 2>();
      else if (g + 2 < total)
        wait_vm<G::OPS>();
      else
        wait_vm<0>();
      lds_barrier();  // stage g + 1 landed everywhere
    } else {
      wait_vm<0>();  // the last stage: the shared-threshold keys of the last tile
      lds_barrier();
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      mf(F1, i);
      if (read_next && i < 6) {  // (stale but in-bounds after the last stage)
        rd(nxt, 0, 2 * i, F0);
        rd(nxt, 0, 2 * i + 1, F0);
      }
      if (more && i >= G::DMA_SLOT0 && i < G::DMA_SLOT0 + 4) dma_part(fill, 4 + i - G::DMA_SLOT0);
      __builtin_amdgcn_sched_barrier(0);
    }
    if (more) dma_finish();
    // the shared thresholds for this tile's epilogue, read three stages before
    // its end, when every split has published its previous tile: the wait for
    // stage g + 1 of the tile's last stage covers this load (it is issued
    // before the DMA of the stages that wait leaves outstanding)
    if (wave == 1 && ((g + 4) % nk) == 0) dma16(a.gthr + h0 + lane * 4, lds_addr(&ep.tgk[(g / nk) & 1][0]));
    ++g;
  };

  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  using I3 = std::integral_constant<int, 3>;
  using RD = std::true_type;
  using NR = std::false_type;
  for (int ti = 0; ti < nt; ++ti) {
    for (int kt = 0; kt < nk - 4; kt += 4) {
      body(I0{}, RD{});
      body(I1{}, RD{});
      body(I2{}, RD{});
      body(I3{}, RD{});
    }
    body(I0{}, RD{});
    body(I1{}, RD{});
    body(I2{}, RD{});
    body(I3{}, NR{});
    if constexpr (MODE == kWideStore)
      store_tile(ti);
    else
      epilogue(ti);
    if (ti + 1 < nt) {
      init_acc(ti + 1);
#pragma unroll
      for (int u = 0; u < 12; ++u) rd(S0, 0, u, F0);  // the next tile starts on buffer 0
    }
  }

  if constexpr (MODE == kWideStore) return;
  // ---- this split's partial of every row: merge the four holders' statistics
  if constexpr (STATS) {
#pragma unroll
    for (int hb = 0; hb < 4; ++hb) {
      const int rl = wh * 128 + hb * 32 + col;
      ep.u.red[rl][2 * holder + 0] = st_m[hb];
      ep.u.red[rl][2 * holder + 1] = st_s[hb];
    }
    lds_barrier();
  }
  if (h0 + tid < a.N) {
    const size_t row = (size_t)split * a.N + h0 + tid;
    if constexpr (STATS) {
      float M = kStatInit;
#pragma unroll
      for (int i = 0; i < 4; ++i) M = fmaxf(M, ep.u.red[tid][2 * i]);
      float S = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) S += ep.u.red[tid][2 * i + 1] * exp2_fast((ep.u.red[tid][2 * i] - M) * kL2E);
      a.stats[row] = make_float2(M, S);
    }
#pragma unroll
    for (int j = 0; j < KC; ++j)
      if (j >= KC - k)
        a.lists[row * k + (j - (KC - k))] =
            make_int2(__float_as_int(key2f((uint32_t)(lkey[j] >> 32))), (int)~(uint32_t)lkey[j]);
  }
}

template <int KC, int MODE = kWideKBest>
hipError_t launch_k1_wide_kc(dim3 grid, const K1Args& a, hipStream_t st) {
  k1_wide<KC, MODE><<<grid, dim3(256), 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace kb
