// Decoder stand-in of the synthetic decode loop.  Not part of the output
// layer: the method leaves the decoder (an RNN in the paper) outside the
// step, and the loop that measures mini-batching (Section 2.1, Algorithm 2)
// replaces it by a seeded table of states and a drawn length per sentence.
// These kernels keep that bookkeeping on the device so that a loop step
// costs a handful of launches:
//   * standin_alive: entry s*k + r of the batch stays unless its sentence
//     reaches its drawn length this step (every continuation ends together);
//   * standin_next_h: the next step's state of each surviving entry, read
//     from the table at (original sentence id, step, beam slot);
//   * standin_step: the mask, the compaction over it (K3's scan), the
//     gathers of the surviving entries' scores and sentences' ids and,
//     optionally, of their next states, in one launch: a loop step is then
//     the output layer and this.
#include <algorithm>

#include "k3_scan.hpp"

namespace kb {

__global__ __launch_bounds__(256) void standin_alive(int S, const int32_t* __restrict__ S_dev, int k, int t,
                                                     const int32_t* __restrict__ sid,
                                                     const int32_t* __restrict__ lengths,
                                                     uint8_t* __restrict__ alive) {
  const int n = S * k;
  const int live = S_dev ? min(S, *S_dev) : S;  // sentences past it do not exist this step
  for (int e = blockIdx.x * 256 + threadIdx.x; e < n; e += gridDim.x * 256) {
    const int s = e / k;
    alive[e] = (s < live && t < lengths[sid[s]] - 1) ? 1 : 0;
  }
}

template <class V>
__global__ __launch_bounds__(256) void standin_next_h(int n_max, const int32_t* __restrict__ n_dev, int k, int T,
                                                      int t, const int32_t* __restrict__ keep,
                                                      const int32_t* __restrict__ sid, const V* __restrict__ table,
                                                      V* __restrict__ out, int row_words) {
  const int n = n_dev ? min(n_max, *n_dev) : n_max;
  const long long total = (long long)n * row_words;
  for (long long i = (long long)blockIdx.x * 256 + threadIdx.x; i < total; i += (long long)gridDim.x * 256) {
    const int r = (int)(i / row_words);
    const int w = (int)(i - (long long)r * row_words);
    const int e = keep[r];
    const long long src = ((long long)sid[e / k] * T + t) * k + e % k;
    out[i] = table[src * row_words + w];
  }
}

// One step's bookkeeping.  Workgroup 0 writes the compaction's outputs
// (surviving entries and their scores, new offsets, surviving sentences'
// ids, the counts, optionally the mask).  With next_h, every workgroup also
// gathers its share of the surviving entries' next states from the table;
// each works the compaction out again for itself (a scan over the S*k entries
// into its LDS), so no workgroup waits for another and the step's
// bookkeeping is one launch.
template <class V>
__global__ __launch_bounds__(K3_T) void standin_step(int S, const int32_t* __restrict__ S_dev, int k, int t,
                                                     const int32_t* __restrict__ sid,
                                                     const int32_t* __restrict__ lengths,
                                                     const float* __restrict__ score, int32_t* __restrict__ keep,
                                                     int32_t* __restrict__ counts, int32_t* __restrict__ new_off,
                                                     float* __restrict__ prev_next, int32_t* __restrict__ sid_next,
                                                     uint8_t* __restrict__ alive, int32_t* __restrict__ counts_host,
                                                     const V* __restrict__ table, int T, V* __restrict__ next_h,
                                                     int row_words) {
  __shared__ int wsum[K3_W];
  extern __shared__ int keep_l[];  // [S*k] the surviving entries, then [S] the sentences' ids (with next_h only)
  int* const sid_l = keep_l + S * k;
  const int tid = threadIdx.x;
  const bool lead = blockIdx.x == 0;
  const int live = S_dev ? min(S, *S_dev) : S;  // sentences past it do not exist this step
  // sid[s] (inside the array for every s < S) is read without waiting for the
  // device count, so both loads are in flight together; an id is used (to
  // index lengths) only below the count
  auto is_alive = [&](int e) {
    const int s = e / k;
    const int id = s < S ? sid[s] : 0;
    return s < live && t < lengths[id] - 1;
  };
  if (next_h)  // the live sentences' ids, for the state gather
    for (int s = tid; s < S; s += K3_T) sid_l[s] = sid[s];
  const int kept = compact_entries_pass(S * k, is_alive, [&](int o, int e) {
    if (lead) {
      keep[o] = e;
      prev_next[o] = score[e];
    }
    if (next_h) keep_l[o] = e;
  }, wsum);
  if (lead) {
    int sbase, ebase;
    compact_sentences_pass(S, k, is_alive, [&](int pos, int s, int first) {
      new_off[pos] = first;
      sid_next[pos] = sid[s];
    }, wsum, sbase, ebase);
    for (int s = sbase + tid; s <= S; s += K3_T) new_off[s] = ebase;  // empty sentences past the survivors
    if (alive)
      for (int e = tid; e < S * k; e += K3_T) alive[e] = is_alive(e) ? 1 : 0;
    if (tid == 0) {
      counts[0] = kept;
      counts[1] = sbase;
      if (counts_host) {
        // pinned host memory: the counts, then the step's tag t + 1, each
        // pushed out by a system-scope fence, so a host that sees the tag sees
        // the counts (before the kernel has completed)
        counts_host[0] = kept;
        counts_host[1] = sbase;
        __threadfence_system();
        counts_host[2] = t + 1;
        __threadfence_system();
      }
    }
  }
  if (next_h) {
    __syncthreads();  // keep_l and sid_l complete
    // this workgroup's surviving rows: an even share of the S*k the launch was
    // sized for among the workgroups past the first (which did the bookkeeping),
    // or all of them when it is alone
    const int G = (int)gridDim.x > 1 ? (int)gridDim.x - 1 : 1;
    const int b = (int)gridDim.x > 1 ? (int)blockIdx.x - 1 : 0;
    if (b >= 0) {
      const int per = (S * k + G - 1) / G;
      const int r0 = min(b * per, kept), r1 = min(r0 + per, kept);
      for (int i = r0 * row_words + tid; i < r1 * row_words; i += K3_T) {
        const int r = i / row_words, w = i - r * row_words;
        const int e = keep_l[r];
        const long long src = ((long long)sid_l[e / k] * T + t + 1) * k + e % k;
        next_h[i] = table[src * row_words + w];
      }
    }
  }
}

hipError_t launch_standin_alive(int S, const int32_t* S_dev, int k, int t, const int32_t* sid, const int32_t* lengths,
                                uint8_t* alive, hipStream_t st) {
  const int n = S * k;
  const int blocks = n > 0 ? min((n + 255) / 256, 1024) : 1;
  standin_alive<<<dim3(blocks), dim3(256), 0, st>>>(S, S_dev, k, t, sid, lengths, alive);
  return hipGetLastError();
}

hipError_t launch_standin_next_h(int n_max, const int32_t* n_dev, int k, int T, int t, const int32_t* keep,
                                 const int32_t* sid, const void* table, void* out, size_t row_bytes,
                                 hipStream_t st) {
  const bool v16 = (row_bytes % 16 == 0) && ((uintptr_t)table % 16 == 0) && ((uintptr_t)out % 16 == 0);
  const size_t words = v16 ? row_bytes / 16 : row_bytes / 4;
  const long long total = (long long)n_max * (long long)words;
  int blocks = (int)((total + 255) / 256);
  blocks = blocks < 1 ? 1 : (blocks > 8192 ? 8192 : blocks);
  if (v16)
    standin_next_h<uint4><<<dim3(blocks), dim3(256), 0, st>>>(n_max, n_dev, k, T, t, keep, sid,
                                                              (const uint4*)table, (uint4*)out, (int)words);
  else
    standin_next_h<uint32_t><<<dim3(blocks), dim3(256), 0, st>>>(n_max, n_dev, k, T, t, keep, sid,
                                                                 (const uint32_t*)table, (uint32_t*)out,
                                                                 (int)words);
  return hipGetLastError();
}

// The fused gather keeps the surviving entries and the sentences' ids in LDS:
// at most this many bytes of them.
constexpr long long kStandinFusedLds = 64 * 1024;

hipError_t launch_standin_step(int S, const int32_t* S_dev, int k, int t, const int32_t* sid, const int32_t* lengths,
                               const float* score, int32_t* keep, int32_t* counts, int32_t* new_off,
                               float* prev_next, int32_t* sid_next, uint8_t* alive, int32_t* counts_host,
                               const void* table, int T, void* next_h, size_t row_bytes, hipStream_t st) {
  const long long M = (long long)S * k;
  const bool v16 = (row_bytes % 16 == 0) && ((uintptr_t)table % 16 == 0) && ((uintptr_t)next_h % 16 == 0);
  const long long words = next_h ? (long long)(v16 ? row_bytes / 16 : row_bytes / 4) : 0;
  if (next_h && ((M + S + 1) * (long long)sizeof(int32_t) > kStandinFusedLds || M * words > INT_MAX)) {
    // too many entries for one workgroup's LDS: the bookkeeping, then the gather
    standin_step<uint32_t><<<dim3(1), dim3(K3_T), 0, st>>>(S, S_dev, k, t, sid, lengths, score, keep, counts, new_off,
                                                        prev_next, sid_next, alive, counts_host, nullptr, 0,
                                                        nullptr, 0);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_standin_next_h((int)M, counts, k, T, t + 1, keep, sid, table, next_h, row_bytes, st);
  }
  if (!next_h) {
    standin_step<uint32_t><<<dim3(1), dim3(K3_T), 0, st>>>(S, S_dev, k, t, sid, lengths, score, keep, counts, new_off,
                                                        prev_next, sid_next, alive, counts_host, nullptr, 0,
                                                        nullptr, 0);
    return hipGetLastError();
  }
  // one workgroup per 32 KB of states (at most 256) after the first, which does
  // the bookkeeping: each works out the scan again, which costs little next to
  // its share of the copy
  const long long bytes = M * (long long)row_bytes;
  const int G = 1 + (int)std::min<long long>((bytes + (32 << 10) - 1) >> 15, 255);
  const size_t lds = (size_t)(M + S + 1) * sizeof(int32_t);
  if (lds > 48 * 1024) {
    static bool attr_set[2] = {false, false};  // the LDS ceiling, raised once per process and variant
    if (!attr_set[v16]) {
      const hipError_t e = v16 ? hipFuncSetAttribute(reinterpret_cast<const void*>(&standin_step<uint4>),
                                                     hipFuncAttributeMaxDynamicSharedMemorySize,
                                                     (int)kStandinFusedLds)
                               : hipFuncSetAttribute(reinterpret_cast<const void*>(&standin_step<uint32_t>),
                                                     hipFuncAttributeMaxDynamicSharedMemorySize,
                                                     (int)kStandinFusedLds);
      if (e != hipSuccess) return e;
      attr_set[v16] = true;
    }
  }
  if (v16)
    standin_step<uint4><<<dim3(G), dim3(K3_T), lds, st>>>(S, S_dev, k, t, sid, lengths, score, keep, counts, new_off,
                                                         prev_next, sid_next, alive, counts_host,
                                                         (const uint4*)table, T, (uint4*)next_h, (int)words);
  else
    standin_step<uint32_t><<<dim3(G), dim3(K3_T), lds, st>>>(S, S_dev, k, t, sid, lengths, score, keep, counts,
                                                            new_off, prev_next, sid_next, alive, counts_host,
                                                            (const uint32_t*)table, T, (uint32_t*)next_h,
                                                            (int)words);
  return hipGetLastError();
}

}  // namespace kb
