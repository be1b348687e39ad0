// Shared device helpers and the host<->kernel argument blocks of libkbest.
#pragma once

#include <hip/hip_runtime.h>

#include <float.h>
#include <limits.h>
#include <stddef.h>
#include <stdint.h>

namespace kb {

constexpr int kWave = 64;
constexpr float kL2E = 1.4426950408889634f;  // log2(e): exp(x) = exp2(x * log2 e)
constexpr float kNoThr = -FLT_MAX;           // "no threshold yet": every finite score passes
constexpr float kStatInit = -1e30f;          // running max before the first score

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// Total order of (score, index) pairs used everywhere: higher score first,
// equal scores keep the lower index (the strict '>' scans of the paper).
__device__ __forceinline__ bool better(float a, int ia, float b, int ib) {
  return a > b || (a == b && ia < ib);
}

__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// Workgroup barrier for LDS only: waits for this wave's LDS operations, not
// for its outstanding global->LDS DMA (a __syncthreads() fence would drain
// the whole DMA ring).  The memory clobber keeps the compiler from moving
// memory accesses across it.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// LDS byte address of a __shared__ object.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// One global->LDS DMA wave-instruction (gfx950 global_load_lds_dwordx4): lane
// i copies 16 bytes from its global address to LDS byte lds_base + 16 * i
// (lds_base wave-uniform, in M0).  Issued from inline assembly so that the
// compiler does not insert its own (conservative) waits for it; callers wait
// with s_waitcnt vmcnt before reading the data.  One wait state after M0.
__device__ __forceinline__ void dma16(const void* g, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g),
               "s"(__builtin_amdgcn_readfirstlane(lds_base))
               : "m0");
}

// ---------------------------------------------------------------- K1
struct K1Args {
  const void* h;      // N x H
  const void* W;      // H x V
  const float* b;     // V
  int N, H, V, k;
  int tps;            // vocabulary tiles per split
  int n_vtiles;       // vocabulary tiles in total
  int vec_ok;         // 16-byte vector loads valid for h and W
  float2* stats;      // [P][N]   (max, sum of exp(x - max)) of each split
  int2* lists;        // [P][N][k] (score bits, word) of each split, best first
  uint32_t* gthr;     // [row_tiles * BH] shared per-row threshold keys (order-preserving), zeroed per call
  uint32_t* gmax;     // [16][row_tiles * BH] running-max keys of splits 0..15 per row (split-major:
                      // a wave's updates and reads touch 64 consecutive rows), zeroed per call
                      // (256 x 256 tile kernel only)
  int row_tiles;      // R
  int P;              // vocabulary splits
  int grp;            // row tiles per XCD group
  int no_stats;       // 1: the statistics may be skipped (greedy argmax; only the
                      //    256 x 256 tile kernel, k = 1, uses it)
  int share;          // 1: rows' thresholds are shared through gthr; 0: gthr is neither
                      //    read nor written (the other tiles' kernels; the 256 x 256 one
                      //    always shares)
  float* logits;      // N x V scores p = W h (the unfused baseline's projection only)
};

// Workgroup -> (row tile, split).  Workgroups are dealt to the 8 XCDs
// round-robin by block index; block b lands on XCD b % 8.  Each XCD is given
// a contiguous run of cells of an ordering in which groups of `grp` row tiles
// are walked split by split, so one XCD's L2 holds a few row tiles of h and
// sees each W tile requested by all of them at about the same time.
__device__ __forceinline__ void k1_cell(const K1Args& a, int b, int& row_tile, int& split) {
  const int T = a.row_tiles * a.P;
  const int x = b & 7, j = b >> 3;
  const int c = x * (T >> 3) + min(x, T & 7) + j;
  const int full = a.row_tiles / a.grp;            // complete row groups
  const int gcells = a.grp * a.P;
  int rg = c / gcells, gr = a.grp, q = c - rg * gcells;
  if (rg >= full) {                                // the last, smaller group
    gr = a.row_tiles - full * a.grp;
    rg = full;
    q = c - full * gcells;
  }
  split = q / gr;
  row_tile = rg * a.grp + (q - split * gr);
}

// Tile shapes of the fused projection kernel.
enum K1Layout { K1_L256 = 0, K1_L128 = 1, K1_L32 = 2, K1_W256 = 3, K1_L32M = 4, K1_L32S = 5, K1_L64 = 6 };

// dma: the LDS-DMA pipeline (bf16, H % 128 == 0, V % 8 == 0, 16-byte aligned h and W);
// layout K1_W256 (256 x 256 tiles) exists only with it.
hipError_t launch_k1(int bf16, int dma, int layout, int kc, dim3 grid, const K1Args& a, hipStream_t st);
hipError_t launch_zero_u32(uint32_t* p, int n, hipStream_t st);

}  // namespace kb
