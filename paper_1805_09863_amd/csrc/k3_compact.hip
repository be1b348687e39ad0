// K3: stable removal of finished hypotheses from the batch (Section 2.1,
// Algorithm 2), and the row gather that moves the survivors' state.
//
// One 1024-thread workgroup walks the S*k entries in chunks: per-thread
// counts, a workgroup exclusive scan (wave shuffles, then the 16 wave totals),
// and each survivor writes its index at its rank.  A second pass does the same
// over sentences with a packed (surviving sentence, surviving entries) count
// to build the new offsets.  Integer work only: results are exact.
#include "k3_scan.hpp"

namespace kb {

__global__ __launch_bounds__(K3_T) void k3_compact(int S, int k, const uint8_t* __restrict__ alive,
                                                   int32_t* __restrict__ keep, int32_t* __restrict__ kept_count,
                                                   int32_t* __restrict__ new_off, int32_t* __restrict__ kept_sent,
                                                   int32_t* __restrict__ new_S) {
  __shared__ int wsum[K3_W];
  const int tid = threadIdx.x;
  auto is_alive = [&](int e) { return alive[e] != 0; };
  const int kept = compact_entries_pass(S * k, is_alive, [&](int o, int e) { keep[o] = e; }, wsum);
  if (tid == 0) *kept_count = kept;

  if (new_off == nullptr && kept_sent == nullptr && new_S == nullptr) return;
  int sbase, ebase;
  compact_sentences_pass(S, k, is_alive, [&](int pos, int s, int first) {
    if (kept_sent) kept_sent[pos] = s;
    if (new_off) new_off[pos] = first;
  }, wsum, sbase, ebase);
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

// ---------------------------------------------------------------- M-entry compaction
// The batch as a flat list of M entries, each tagged (optionally) with its
// sentence; sentence ids never decrease along the list.  keep_idx is the
// stable list of surviving entries; a sentence survives if any of its entries
// does, and its new offset is the position of its first surviving entry.

namespace kb {

constexpr int KE_ITEMS = 4;
constexpr int KE_BLOCK = K3_T * KE_ITEMS;  // entries per workgroup of the multi-workgroup form

// One workgroup (M <= KE_ONE): surviving entries first (their list also kept
// in LDS), then over the kept positions the first entry of every sentence.
__global__ __launch_bounds__(K3_T) void k3_compact_entries(int M, const uint8_t* __restrict__ alive,
                                                           int32_t* __restrict__ keep, int32_t* __restrict__ kept_count,
                                                           const int32_t* __restrict__ es, int32_t* __restrict__ new_off,
                                                           int32_t* __restrict__ new_S) {
  __shared__ int wsum[K3_W];
  __shared__ int skeep[KE_ONE];
  const int tid = threadIdx.x;
  int base = 0;
  for (int c0 = 0; c0 < M; c0 += KE_BLOCK) {
    const int i0 = c0 + tid * KE_ITEMS;
    int f[KE_ITEMS];
    int lc = 0;
#pragma unroll
    for (int e = 0; e < KE_ITEMS; ++e) {
      f[e] = (i0 + e < M) ? (alive[i0 + e] != 0) : 0;
      lc += f[e];
    }
    int total;
    int o = base + block_excl_scan(lc, wsum, &total);
#pragma unroll
    for (int e = 0; e < KE_ITEMS; ++e)
      if (f[e]) {
        keep[o] = i0 + e;
        skeep[o] = i0 + e;
        ++o;
      }
    base += total;
  }
  if (tid == 0) *kept_count = base;
  if (new_off == nullptr && new_S == nullptr) return;  // es is given whenever they are and M > 0
  __syncthreads();  // skeep complete
  const int kept = base;
  int nb = 0;
  for (int p0 = 0; p0 < kept; p0 += KE_BLOCK) {
    const int q0 = p0 + tid * KE_ITEMS;
    int f[KE_ITEMS];
    int lc = 0;
#pragma unroll
    for (int e = 0; e < KE_ITEMS; ++e) {
      const int p = q0 + e;
      f[e] = p < kept && (p == 0 || es[skeep[p - 1]] != es[skeep[p]]);
      lc += f[e];
    }
    int total;
    int o = nb + block_excl_scan(lc, wsum, &total);
#pragma unroll
    for (int e = 0; e < KE_ITEMS; ++e)
      if (f[e]) {
        if (new_off) new_off[o] = q0 + e;
        ++o;
      }
    nb += total;
  }
  if (tid == 0) {
    if (new_off) new_off[nb] = kept;
    if (new_S) *new_S = nb;
  }
}

// Multi-workgroup form: count per workgroup, scan the counts, scatter.  Pass
// 0 flags the surviving entries; pass 1 flags the kept positions that start a
// sentence (read from the keep list pass 0 wrote).
template <int PASS>
__device__ __forceinline__ int ke_flag(int i, int M, const uint8_t* alive, const int32_t* keep, int kept,
                                       const int32_t* es) {
  if (PASS == 0) return i < M ? (alive[i] != 0) : 0;
  return i < kept ? (i == 0 || es[keep[i - 1]] != es[keep[i]]) : 0;
}

template <int PASS>
__global__ __launch_bounds__(K3_T) void ke_count(int M, const uint8_t* __restrict__ alive,
                                                 const int32_t* __restrict__ keep, const int32_t* __restrict__ kept_dev,
                                                 const int32_t* __restrict__ es, int32_t* __restrict__ cnt) {
  __shared__ int wsum[K3_W];
  const int kept = PASS ? *kept_dev : 0;
  const int i0 = blockIdx.x * KE_BLOCK + threadIdx.x * KE_ITEMS;
  int lc = 0;
#pragma unroll
  for (int e = 0; e < KE_ITEMS; ++e) lc += ke_flag<PASS>(i0 + e, M, alive, keep, kept, es);
  int total;
  block_excl_scan(lc, wsum, &total);
  if (threadIdx.x == 0) cnt[blockIdx.x] = total;
}

// exclusive scan of nb counts in place; the total to tot (and out, if given)
__global__ __launch_bounds__(K3_T) void ke_scan(int nb, int32_t* __restrict__ cnt, int32_t* __restrict__ tot,
                                                int32_t* __restrict__ out) {
  __shared__ int wsum[K3_W];
  int base = 0;
  for (int c0 = 0; c0 < nb; c0 += K3_T) {
    const int i = c0 + threadIdx.x;
    const int v = i < nb ? cnt[i] : 0;
    int total;
    const int ex = block_excl_scan(v, wsum, &total);
    if (i < nb) cnt[i] = base + ex;
    base += total;
  }
  if (threadIdx.x == 0) {
    *tot = base;
    if (out) *out = base;
  }
}

// pass 0: keep[rank] = entry; pass 1: new_off[rank] = position, and
// new_off[sentences] = kept
template <int PASS>
__global__ __launch_bounds__(K3_T) void ke_scatter(int M, const uint8_t* __restrict__ alive,
                                                   const int32_t* __restrict__ keep, const int32_t* __restrict__ kept_dev,
                                                   const int32_t* __restrict__ es, const int32_t* __restrict__ prefix,
                                                   const int32_t* __restrict__ nS_dev, int32_t* __restrict__ dst) {
  __shared__ int wsum[K3_W];
  const int kept = PASS ? *kept_dev : 0;
  const int i0 = blockIdx.x * KE_BLOCK + threadIdx.x * KE_ITEMS;
  int f[KE_ITEMS];
  int lc = 0;
#pragma unroll
  for (int e = 0; e < KE_ITEMS; ++e) {
    f[e] = ke_flag<PASS>(i0 + e, M, alive, keep, kept, es);
    lc += f[e];
  }
  int total;
  int o = prefix[blockIdx.x] + block_excl_scan(lc, wsum, &total);
#pragma unroll
  for (int e = 0; e < KE_ITEMS; ++e)
    if (f[e]) dst[o++] = i0 + e;
  if (PASS == 1 && blockIdx.x == 0 && threadIdx.x == 0) dst[*nS_dev] = kept;
}

size_t compact_entries_ws_bytes(int M) {
  if (M <= KE_ONE) return 0;
  const size_t nb = ((size_t)M + KE_BLOCK - 1) / KE_BLOCK;
  return ((2 * nb + 2) * sizeof(int32_t) + 255) / 256 * 256;
}

hipError_t launch_compact_entries(int M, const uint8_t* alive, int32_t* keep, int32_t* kept_count, const int32_t* es,
                                  int32_t* new_off, int32_t* new_S, void* ws, hipStream_t st) {
  if (M <= KE_ONE) {
    k3_compact_entries<<<dim3(1), dim3(K3_T), 0, st>>>(M, alive, keep, kept_count, es, new_off, new_S);
    return hipGetLastError();
  }
  const int nb = (M + KE_BLOCK - 1) / KE_BLOCK;
  int32_t* cnt0 = static_cast<int32_t*>(ws);
  int32_t* cnt1 = cnt0 + nb;
  int32_t* tot = cnt1 + nb;  // [0] kept, [1] surviving sentences
  ke_count<0><<<dim3(nb), dim3(K3_T), 0, st>>>(M, alive, nullptr, nullptr, nullptr, cnt0);
  ke_scan<<<dim3(1), dim3(K3_T), 0, st>>>(nb, cnt0, tot, kept_count);
  ke_scatter<0><<<dim3(nb), dim3(K3_T), 0, st>>>(M, alive, nullptr, nullptr, nullptr, cnt0, nullptr, keep);
  if (new_off == nullptr && new_S == nullptr) return hipGetLastError();
  ke_count<1><<<dim3(nb), dim3(K3_T), 0, st>>>(M, nullptr, keep, tot, es, cnt1);
  ke_scan<<<dim3(1), dim3(K3_T), 0, st>>>(nb, cnt1, tot + 1, new_S);
  if (new_off)
    ke_scatter<1><<<dim3(nb), dim3(K3_T), 0, st>>>(M, nullptr, keep, tot, es, cnt1, tot + 1, new_off);
  return hipGetLastError();
}

// ---------------------------------------------------------------- KB_DEBUG checks
// Device-resident index arrays are trusted by the kernels; with KB_DEBUG set
// the host runs these first and reads the flag word back (0 = valid).

// sentence offsets: bit 0 off[0] != 0, bit 1 some off[s + 1] < off[s],
// bit 2 off[S] > N
__global__ __launch_bounds__(256) void check_offsets(int S, int N, const int32_t* __restrict__ off,
                                                     int32_t* __restrict__ flag) {
  __shared__ int bad;
  if (threadIdx.x == 0) bad = 0;
  __syncthreads();
  int b = 0;
  if (threadIdx.x == 0) {
    if (off[0] != 0) b |= 1;
    if (off[S] > N) b |= 4;
  }
  for (int s = threadIdx.x; s < S; s += 256)
    if (off[s + 1] < off[s]) b |= 2;
  if (b) atomicOr(&bad, b);
  __syncthreads();
  if (threadIdx.x == 0) *flag = bad;
}

// entry sentence ids: bit 0 es[0] < 0, bit 1 some es[i + 1] < es[i]
__global__ __launch_bounds__(256) void check_sorted(int M, const int32_t* __restrict__ es, int32_t* __restrict__ flag) {
  __shared__ int bad;
  if (threadIdx.x == 0) bad = 0;
  __syncthreads();
  int b = 0;
  if (threadIdx.x == 0 && M > 0 && es[0] < 0) b |= 1;
  for (int i = threadIdx.x; i + 1 < M; i += 256)
    if (es[i + 1] < es[i]) b |= 2;
  if (b) atomicOr(&bad, b);
  __syncthreads();
  if (threadIdx.x == 0) *flag = bad;
}

hipError_t launch_check_offsets(int S, int N, const int32_t* off, int32_t* flag, hipStream_t st) {
  check_offsets<<<dim3(1), dim3(256), 0, st>>>(S, N, off, flag);
  return hipGetLastError();
}

hipError_t launch_check_sorted(int M, const int32_t* es, int32_t* flag, hipStream_t st) {
  check_sorted<<<dim3(1), dim3(256), 0, st>>>(M, es, flag);
  return hipGetLastError();
}

}  // namespace kb
