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
  uint32_t* gthr;     // [N] shared per-row threshold (order-preserving key), zeroed per call
};

// Tile shapes of the fused projection kernel.
enum K1Layout { K1_L256 = 0, K1_L128 = 1, K1_L32 = 2 };

// dma: the LDS-DMA pipeline (bf16, H % 32 == 0, V % 8 == 0, 16-byte aligned h and W)
hipError_t launch_k1(int bf16, int dma, int layout, int kc, dim3 grid, const K1Args& a, hipStream_t st);
hipError_t launch_zero_u32(uint32_t* p, int n, hipStream_t st);

// ---------------------------------------------------------------- K2
struct K2Args {
  const float2* stats;
  const int2* lists;
  int P, N, V, k, S;
  const float* prev;
  const int32_t* off;
  int32_t* tok;
  int32_t* par;
  float* score;
  float* row_lse;     // nullable
};

hipError_t launch_k2(const K2Args& a, hipStream_t st);

// ---------------------------------------------------------------- K3 / gather
hipError_t launch_compact(int S, int k, const uint8_t* alive, int32_t* keep, int32_t* kept_count,
                          int32_t* new_off, int32_t* kept_sent, int32_t* new_S, hipStream_t st);

hipError_t launch_gather(int n_max, const int32_t* n_dev, const int32_t* idx, const void* src,
                         void* dst, size_t row_bytes, hipStream_t st);

}  // namespace kb
