// The one-workgroup compaction scan of K3 (stable removal of finished
// entries, Section 2.1, Algorithm 2), written once for every kernel that
// compacts an S x k batch: kb_compact_beams's kernel and the decoder
// stand-in's fused step.  What makes an entry survive, and what is written
// for each survivor and each surviving sentence, are the caller's.
#pragma once

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

// Entry pass over the S*k entries in chunks (per-thread counts, workgroup
// exclusive scan, each survivor at its rank): on_entry(rank, entry).  Returns
// the number of survivors (every thread gets it).
template <class Alive, class OnEntry>
__device__ __forceinline__ int compact_entries_pass(int M, Alive alive, OnEntry on_entry, int* wsum) {
  const int tid = threadIdx.x;
  int base = 0;
  for (int c0 = 0; c0 < M; c0 += K3_T * K3_ITEMS) {
    const int i0 = c0 + tid * K3_ITEMS;
    int f[K3_ITEMS];
    int lc = 0;
#pragma unroll
    for (int e = 0; e < K3_ITEMS; ++e) {
      f[e] = (i0 + e < M) ? (alive(i0 + e) ? 1 : 0) : 0;
      lc += f[e];
    }
    int total;
    int o = base + block_excl_scan(lc, wsum, &total);
#pragma unroll
    for (int e = 0; e < K3_ITEMS; ++e)
      if (f[e]) on_entry(o++, i0 + e);
    base += total;
  }
  return base;
}

// Sentence pass: a sentence survives if any of its k entries does; its rank
// among the survivors and the position of its first surviving entry are
// scanned together as one packed count ((survives << 20) | surviving entries,
// so S * k < 2^20 per chunk of K3_T sentences): on_sentence(rank, sentence,
// first entry).  Returns (survivors, their entries) in sents / ents.
template <class Alive, class OnSentence>
__device__ __forceinline__ void compact_sentences_pass(int S, int k, Alive alive, OnSentence on_sentence, int* wsum,
                                                       int& sents, int& ents) {
  const int tid = threadIdx.x;
  int sbase = 0, ebase = 0;
  for (int s0 = 0; s0 < S; s0 += K3_T) {
    const int s = s0 + tid;
    int cnt = 0;
    if (s < S)
      for (int j = 0; j < k; ++j) cnt += alive(s * k + j) ? 1 : 0;
    const int flag = cnt > 0;
    int total;
    const int ex = block_excl_scan(cnt | (flag << 20), wsum, &total);
    if (flag) on_sentence(sbase + (ex >> 20), s, ebase + (ex & 0xFFFFF));
    sbase += total >> 20;
    ebase += total & 0xFFFFF;
  }
  sents = sbase;
  ents = ebase;
}

}  // namespace kb
