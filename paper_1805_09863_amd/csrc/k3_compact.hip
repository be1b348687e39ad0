// K3: stable removal of finished hypotheses from the batch (Section 2.1,
// Algorithm 2), and the row gather that moves the survivors' state.
//
// One 1024-thread workgroup walks the S*k entries in chunks: per-thread
// counts, a workgroup exclusive scan (wave shuffles, then the 16 wave totals),
// and each survivor writes its index at its rank.  A second pass does the same
// over sentences with a packed (surviving sentence, surviving entries) count
// to build the new offsets.  Integer work only: results are exact.
#include "kb_launch.hpp"

namespace kb {

constexpr int K3_T = 1024;
constexpr int K3_W = K3_T / 64;
constexpr int K3_ITEMS = 4;

// Exclusive scan of v over the workgroup; returns the total in *total.
__device__ __forceinline__ int block_excl_scan(int v, int* wsum, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int y = __shfl_up(x, d, 64);
    if (lane >= d) x += y;
  }
  __syncthreads();  // wsum is reused between calls
  if (lane == 63) wsum[wave] = x;
  __syncthreads();
  int before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < K3_W; ++w) {
    const int t = wsum[w];
    before += (w < wave) ? t : 0;
    all += t;
  }
  *total = all;
  return before + x - v;
}

__global__ __launch_bounds__(K3_T) void k3_compact(int S, int k, const uint8_t* __restrict__ alive,
                                                   int32_t* __restrict__ keep, int32_t* __restrict__ kept_count,
                                                   int32_t* __restrict__ new_off, int32_t* __restrict__ kept_sent,
                                                   int32_t* __restrict__ new_S) {
  __shared__ int wsum[K3_W];
  const int tid = threadIdx.x;
  const int M = S * k;

  int base = 0;
  for (int c0 = 0; c0 < M; c0 += K3_T * K3_ITEMS) {
    const int i0 = c0 + tid * K3_ITEMS;
    int f[K3_ITEMS];
    int lc = 0;
#pragma unroll
    for (int e = 0; e < K3_ITEMS; ++e) {
      f[e] = (i0 + e < M) ? (alive[i0 + e] != 0) : 0;
      lc += f[e];
    }
    int total;
    int o = base + block_excl_scan(lc, wsum, &total);
#pragma unroll
    for (int e = 0; e < K3_ITEMS; ++e)
      if (f[e]) keep[o++] = i0 + e;
    base += total;
  }
  if (tid == 0) *kept_count = base;

  if (new_off == nullptr && kept_sent == nullptr && new_S == nullptr) return;
  // per sentence: (survives << 20) | surviving entries, scanned together
  int sbase = 0, ebase = 0;
  for (int s0 = 0; s0 < S; s0 += K3_T) {
    const int s = s0 + tid;
    int cnt = 0;
    if (s < S)
      for (int j = 0; j < k; ++j) cnt += (alive[(size_t)s * k + j] != 0);
    const int flag = cnt > 0;
    int total;
    const int ex = block_excl_scan(cnt | (flag << 20), wsum, &total);
    if (flag) {
      const int pos = sbase + (ex >> 20);
      if (kept_sent) kept_sent[pos] = s;
      if (new_off) new_off[pos] = ebase + (ex & 0xFFFFF);
    }
    sbase += total >> 20;
    ebase += total & 0xFFFFF;
  }
  // the end of the last surviving sentence, repeated up to entry S: a launch
  // sized for more sentences than survive sees only empty ones past new_S
  if (new_off)
    for (int s = sbase + tid; s <= S; s += K3_T) new_off[s] = ebase;
  if (tid == 0 && new_S) *new_S = sbase;
}

hipError_t launch_compact(int S, int k, const uint8_t* alive, int32_t* keep, int32_t* kept_count,
                          int32_t* new_off, int32_t* kept_sent, int32_t* new_S, hipStream_t st) {
  k3_compact<<<dim3(1), dim3(K3_T), 0, st>>>(S, k, alive, keep, kept_count, new_off, kept_sent, new_S);
  return hipGetLastError();
}

// ---------------------------------------------------------------- gather
template <class V>
__global__ __launch_bounds__(256) void gather_rows(int n_max, const int32_t* __restrict__ n_dev,
                                                   const int32_t* __restrict__ idx, const V* __restrict__ src,
                                                   V* __restrict__ dst, int row_words) {
  const int n = n_dev ? min(n_max, *n_dev) : n_max;
  const long long total = (long long)n * row_words;
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (long long)gridDim.x * blockDim.x) {
    const long long r = i / row_words;
    const int w = (int)(i - r * row_words);
    dst[i] = src[(long long)idx[r] * row_words + w];
  }
}

hipError_t launch_gather(int n_max, const int32_t* n_dev, const int32_t* idx, const void* src, void* dst,
                         size_t row_bytes, hipStream_t st) {
  const bool v16 = (row_bytes % 16 == 0) && ((uintptr_t)src % 16 == 0) && ((uintptr_t)dst % 16 == 0);
  const size_t words = v16 ? row_bytes / 16 : row_bytes / 4;
  const long long total = (long long)n_max * (long long)words;
  int blocks = (int)((total + 255) / 256);
  blocks = blocks < 1 ? 1 : (blocks > 8192 ? 8192 : blocks);
  if (v16)
    gather_rows<uint4><<<dim3(blocks), dim3(256), 0, st>>>(n_max, n_dev, idx, (const uint4*)src, (uint4*)dst,
                                                           (int)words);
  else
    gather_rows<uint32_t><<<dim3(blocks), dim3(256), 0, st>>>(n_max, n_dev, idx, (const uint32_t*)src,
                                                              (uint32_t*)dst, (int)words);
  return hipGetLastError();
}

}  // namespace kb
