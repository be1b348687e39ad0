// Launchers of the kernels around the projection: the split and beam merge
// (K2), the compaction and gathers (K3), the unfused baseline's stages, the
// per-hypothesis end of sentence and the decoder stand-in.  Kept apart from
// kb_common.hpp, which holds only what the projection kernels compile.
#pragma once

#include "kb_common.hpp"

namespace kb {

// ---------------------------------------------------------------- K1, few rows
// Steps of at most FEW_ROWS live rows, operands 16-byte loadable: VALU
// projection streaming W once (k1_few.hip).  Layout code K1_FEW.
constexpr int FEW_ROWS = 8;
constexpr int K1_FEW = 16;
int few_chunk_words(int bf16);                   // words per chunk (one "tile")
size_t few_lds_needed(int bf16, int N, int H, int tps);  // LDS bytes of a launch (tps chunks per split)
hipError_t launch_k1_few(int bf16, dim3 grid, const K1Args& a, hipStream_t st);

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
hipError_t launch_add_word_base(int2* lists, size_t n, int base, int v_shard, hipStream_t st);
hipError_t launch_k2_argmax(const int2* lists, int P, int N, int32_t* tok, float* val, hipStream_t st);

// ---------------------------------------------------------------- K3 / gather
hipError_t launch_compact(int S, int k, const uint8_t* alive, int32_t* keep, int32_t* kept_count,
                          int32_t* new_off, int32_t* kept_sent, int32_t* new_S, hipStream_t st);

// M-entry form (sentence ids per entry); one workgroup up to KE_ONE entries,
// else three kernels per pass over a workspace of compact_entries_ws_bytes(M)
constexpr int KE_ONE = 16384;
size_t compact_entries_ws_bytes(int M);
hipError_t launch_compact_entries(int M, const uint8_t* alive, int32_t* keep, int32_t* kept_count, const int32_t* es,
                                  int32_t* new_off, int32_t* new_S, void* ws, hipStream_t st);
// KB_DEBUG validation of device-resident index arrays (flag word 0 = valid)
hipError_t launch_check_offsets(int S, int N, const int32_t* off, int32_t* flag, hipStream_t st);
hipError_t launch_check_sorted(int M, const int32_t* es, int32_t* flag, hipStream_t st);

hipError_t launch_gather(int n_max, const int32_t* n_dev, const int32_t* idx, const void* src,
                         void* dst, size_t row_bytes, hipStream_t st);

// ---------------------------------------------------------------- unfused baseline
hipError_t launch_k1_wide_store(dim3 grid, const K1Args& a, hipStream_t st);
hipError_t launch_uf_add_bias(float* x, const float* b, int N, int V, hipStream_t st);
hipError_t launch_uf_softmax3(float* x, int N, int V, float* row_lse, hipStream_t st);
hipError_t launch_uf_kbest_rows(const float* p, int N, int V, int k, float2* stats, int2* lists, hipStream_t st);
hipError_t launch_uf_fused_rows(const float* x, const float* b, int N, int V, int k, float2* stats, int2* lists,
                                hipStream_t st);

// ---------------------------------------------------------------- per-hypothesis EOS
hipError_t launch_beam_finish(int S, int k, int t, int T, int eos, const int32_t* token, const int32_t* parent,
                              const float* score, const int32_t* sid, int32_t* beam, const int32_t* prev_keep,
                              int prev_hist_base, int hist_base, int32_t* hist_token, int32_t* hist_parent,
                              int32_t* fin_count, float* fin_score, int32_t* fin_len, int32_t* fin_hist,
                              uint8_t* alive, hipStream_t st);
hipError_t launch_beam_backtrace(int S0, int k, int T, float alpha, const int32_t* fin_count, const float* fin_score,
                                 const int32_t* fin_len, const int32_t* fin_hist, const int32_t* hist_token,
                                 const int32_t* hist_parent, int32_t* out_tokens, int32_t* out_len,
                                 float* out_score, float* out_norm, hipStream_t st);

// ---------------------------------------------------------------- decoder stand-in
hipError_t launch_standin_alive(int S, const int32_t* S_dev, int k, int t, const int32_t* sid, const int32_t* lengths,
                                uint8_t* alive, hipStream_t st);
hipError_t launch_standin_step(int S, const int32_t* S_dev, int k, int t, const int32_t* sid, const int32_t* lengths,
                               const float* score, int32_t* keep, int32_t* counts, int32_t* new_off,
                               float* prev_next, int32_t* sid_next, uint8_t* alive, int32_t* counts_host,
                               const void* table, int T, void* next_h, size_t row_bytes, hipStream_t st);
hipError_t launch_standin_next_h(int n_max, const int32_t* n_dev, int k, int T, int t, const int32_t* keep,
                                 const int32_t* sid, const void* table, void* out, size_t row_bytes,
                                 hipStream_t st);

}  // namespace kb
