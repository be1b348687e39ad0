// Per-hypothesis end of sentence for the beam search around the output layer
// (Section 2.1, Algorithm 2: every hypothesis that produced EOS leaves the
// batch; a sentence is done when none of its hypotheses is left).
//
// beam_finish, one thread per live sentence s, after a step's k-best:
//   * the sentence's beam is its current size k_s <= k: of its k sorted
//     continuations only the first k_s are taken;
//   * every continuation is recorded in the step's history (token, history
//     id of the parent hypothesis);
//   * a taken continuation whose token is EOS (or any, at the last step T - 1)
//     is finished: it goes to the sentence's finished store (score, length,
//     history id) and the beam shrinks by one; the others stay (alive).
// beam_backtrace, one thread per sentence: the finished hypothesis with the
// best length-normalised score (score / length^alpha; ties: the earlier one)
// and its tokens, read back through the history.
#include "kb_launch.hpp"

namespace kb {

__global__ __launch_bounds__(256) void beam_finish(int S, int k, int t, int T, int eos,
                                                   const int32_t* __restrict__ token,
                                                   const int32_t* __restrict__ parent,
                                                   const float* __restrict__ score,
                                                   const int32_t* __restrict__ sid, int32_t* __restrict__ beam,
                                                   const int32_t* __restrict__ prev_keep, int prev_hist_base,
                                                   int hist_base, int32_t* __restrict__ hist_token,
                                                   int32_t* __restrict__ hist_parent,
                                                   int32_t* __restrict__ fin_count, float* __restrict__ fin_score,
                                                   int32_t* __restrict__ fin_len, int32_t* __restrict__ fin_hist,
                                                   uint8_t* __restrict__ alive) {
  const int s = blockIdx.x * 256 + threadIdx.x;
  if (s >= S) return;
  const int ks = beam[s];
  const int o = sid[s];
  int nf = fin_count[o], left = ks;
  for (int r = 0; r < k; ++r) {
    const int e = s * k + r;
    const int tok = token[e];
    const int p = parent[e];
    hist_token[hist_base + e] = tok;
    hist_parent[hist_base + e] = prev_keep ? prev_hist_base + prev_keep[p] : -1;
    uint8_t keep = 0;
    if (r < ks) {
      if (tok == eos || t + 1 >= T) {
        fin_score[o * k + nf] = score[e];
        fin_len[o * k + nf] = t + 1;
        fin_hist[o * k + nf] = hist_base + e;
        ++nf;
        --left;
      } else {
        keep = 1;
      }
    }
    alive[e] = keep;
  }
  fin_count[o] = nf;
  beam[s] = left;
}

__global__ __launch_bounds__(256) void beam_backtrace(int S0, int k, int T, float alpha,
                                                      const int32_t* __restrict__ fin_count,
                                                      const float* __restrict__ fin_score,
                                                      const int32_t* __restrict__ fin_len,
                                                      const int32_t* __restrict__ fin_hist,
                                                      const int32_t* __restrict__ hist_token,
                                                      const int32_t* __restrict__ hist_parent,
                                                      int32_t* __restrict__ out_tokens, int32_t* __restrict__ out_len,
                                                      float* __restrict__ out_score, float* __restrict__ out_norm) {
  const int s = blockIdx.x * 256 + threadIdx.x;
  if (s >= S0) return;
  const int n = fin_count[s];
  int best = -1;
  float bn = -INFINITY;
  for (int f = 0; f < n; ++f) {
    const float v = fin_score[s * k + f] / powf((float)fin_len[s * k + f], alpha);
    if (best < 0 || v > bn) {
      bn = v;
      best = f;
    }
  }
  int len = 0;
  if (best >= 0) {
    len = fin_len[s * k + best];
    int h = fin_hist[s * k + best];
    for (int pos = len - 1; pos >= 0; --pos) {
      out_tokens[(size_t)s * T + pos] = hist_token[h];
      h = hist_parent[h];
    }
    out_score[s] = fin_score[s * k + best];
    out_norm[s] = bn;
  } else {
    out_score[s] = -INFINITY;
    out_norm[s] = -INFINITY;
  }
  for (int pos = len; pos < T; ++pos) out_tokens[(size_t)s * T + pos] = -1;
  out_len[s] = len;
}

hipError_t launch_beam_finish(int S, int k, int t, int T, int eos, const int32_t* token, const int32_t* parent,
                              const float* score, const int32_t* sid, int32_t* beam, const int32_t* prev_keep,
                              int prev_hist_base, int hist_base, int32_t* hist_token, int32_t* hist_parent,
                              int32_t* fin_count, float* fin_score, int32_t* fin_len, int32_t* fin_hist,
                              uint8_t* alive, hipStream_t st) {
  if (S <= 0) return hipSuccess;
  beam_finish<<<dim3((S + 255) / 256), dim3(256), 0, st>>>(S, k, t, T, eos, token, parent, score, sid, beam,
                                                           prev_keep, prev_hist_base, hist_base, hist_token,
                                                           hist_parent, fin_count, fin_score, fin_len, fin_hist,
                                                           alive);
  return hipGetLastError();
}

hipError_t launch_beam_backtrace(int S0, int k, int T, float alpha, const int32_t* fin_count, const float* fin_score,
                                 const int32_t* fin_len, const int32_t* fin_hist, const int32_t* hist_token,
                                 const int32_t* hist_parent, int32_t* out_tokens, int32_t* out_len,
                                 float* out_score, float* out_norm, hipStream_t st) {
  if (S0 <= 0) return hipSuccess;
  beam_backtrace<<<dim3((S0 + 255) / 256), dim3(256), 0, st>>>(S0, k, T, alpha, fin_count, fin_score, fin_len,
                                                               fin_hist, hist_token, hist_parent, out_tokens,
                                                               out_len, out_score, out_norm);
  return hipGetLastError();
}

}  // namespace kb
