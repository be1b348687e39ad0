// K2: merge the vocabulary splits of every row, then the rows of every sentence.
//
// One workgroup per sentence.  For each of its rows (one wave per row):
//   * LSE = M + ln(sum_p s_p * exp(m_p - M)) over the P split partials -- the
//     rescaling identity of Algorithm 4 applied between shards, the reduction
//     step of Algorithm 6 extended from (max, best) to softmax statistics;
//   * the row's k best words: k rounds of a wave-wide arg-best over the heads
//     of the P sorted split lists (strict total order: higher score, then
//     lower word);
//   * candidate score = prev + x - LSE.
// Rows are taken in chunks; each chunk's candidates and the running k best of
// the sentence are ranked by (score desc, flat index asc), flat index being
// (row - first row) * V + word, and the first k are kept.  Because the score
// adds a per-row constant to x, a sentence's k best lie in the union of its
// rows' k best, so nothing outside these candidates can be selected.
#include "kb_common.hpp"

namespace kb {

constexpr int K2_RC = 16;   // rows per chunk
constexpr int K2_LPL = 4;   // split lists per lane: P <= 256
constexpr int K2_C = K2_RC * 16 + 16;

struct Cand {
  float s;
  int flat;
};

__device__ __forceinline__ bool cbetter(float a, int fa, float b, int fb) { return a > b || (a == b && fa < fb); }

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, __shfl_xor(v, m, 64));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
  return v;
}

__global__ __launch_bounds__(256) void k2_merge(K2Args a) {
  __shared__ float c_s[K2_C];
  __shared__ int c_f[K2_C];
  __shared__ int c_t[K2_C];
  __shared__ int c_p[K2_C];
  __shared__ float n_s[16];
  __shared__ int n_f[16], n_t[16], n_p[16];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int s = blockIdx.x;
  const int k = a.k;
  const int r0 = a.off[s], r1 = a.off[s + 1];

  // running best k of the sentence lives in slots [0, k)
  if (tid < k) {
    c_s[tid] = -INFINITY;
    c_f[tid] = INT_MAX - tid;  // distinct keys for empty slots
    c_t[tid] = -1;
    c_p[tid] = -1;
  }

  for (int cr0 = r0; cr0 < r1; cr0 += K2_RC) {
    const int nrows = min(K2_RC, r1 - cr0);
    for (int ri = wave; ri < nrows; ri += 4) {
      const int r = cr0 + ri;
      float M = kStatInit;
      for (int p = lane; p < a.P; p += 64) M = fmaxf(M, a.stats[(size_t)p * a.N + r].x);
      M = wave_max(M);
      float S = 0.f;
      for (int p = lane; p < a.P; p += 64) {
        const float2 st = a.stats[(size_t)p * a.N + r];
        S += st.y * __expf(st.x - M);
      }
      S = wave_sum(S);
      const float lse = M + __logf(S);
      if (a.row_lse != nullptr && lane == 0) a.row_lse[r] = lse;
      const float base = a.prev[r] - lse;

      int ptr[K2_LPL];
#pragma unroll
      for (int q = 0; q < K2_LPL; ++q) ptr[q] = 0;
      for (int j = 0; j < k; ++j) {
        float bv = -INFINITY;
        int bi = INT_MAX, bq = -1;
#pragma unroll
        for (int q = 0; q < K2_LPL; ++q) {
          const int p = lane + 64 * q;
          if (p < a.P && ptr[q] < k) {
            const int2 e = a.lists[((size_t)p * a.N + r) * k + ptr[q]];
            const float v = __int_as_float(e.x);
            if (better(v, e.y, bv, bi)) {
              bv = v;
              bi = e.y;
              bq = q;
            }
          }
        }
        float wv = bv;
        int wi = bi;
#pragma unroll
        for (int m = 32; m >= 1; m >>= 1) {
          const float ov = __shfl_xor(wv, m, 64);
          const int oi = __shfl_xor(wi, m, 64);
          if (better(ov, oi, wv, wi)) {
            wv = ov;
            wi = oi;
          }
        }
        // the lane whose head won advances that list (entries are unique)
#pragma unroll
        for (int q = 0; q < K2_LPL; ++q)
          if (bq == q && bv == wv && bi == wi) ++ptr[q];
        if (lane == 0) {
          const int slot = k + ri * k + j;
          const bool valid = wv > -INFINITY;
          c_s[slot] = valid ? (wv + base) : -INFINITY;
          c_f[slot] = valid ? (r - r0) * a.V + wi : INT_MAX - slot;
          c_t[slot] = wi;
          c_p[slot] = r;
        }
      }
    }
    __syncthreads();
    // rank every candidate (running best + this chunk) and keep the first k
    const int C = k + nrows * k;
    for (int c = tid; c < C; c += 256) {
      const float sc = c_s[c];
      const int fl = c_f[c];
      int rank = 0;
      for (int o = 0; o < C; ++o) rank += cbetter(c_s[o], c_f[o], sc, fl) ? 1 : 0;
      if (rank < k) {
        n_s[rank] = sc;
        n_f[rank] = fl;
        n_t[rank] = c_t[c];
        n_p[rank] = c_p[c];
      }
    }
    __syncthreads();
    if (tid < k) {
      c_s[tid] = n_s[tid];
      c_f[tid] = n_f[tid];
      c_t[tid] = n_t[tid];
      c_p[tid] = n_p[tid];
    }
    __syncthreads();
  }
  if (tid < k) {
    a.tok[s * k + tid] = c_t[tid];
    a.par[s * k + tid] = c_p[tid];
    a.score[s * k + tid] = c_s[tid];
  }
}

__global__ __launch_bounds__(256) void zero_u32(uint32_t* p, int n) {
  for (int i = blockIdx.x * 256 + threadIdx.x; i < n; i += gridDim.x * 256) p[i] = 0u;
}

hipError_t launch_zero_u32(uint32_t* p, int n, hipStream_t st) {
  const int blocks = n > 0 ? min((n + 255) / 256, 1024) : 1;
  zero_u32<<<dim3(blocks), dim3(256), 0, st>>>(p, n);
  return hipGetLastError();
}

// Greedy (beam 1) merge, the reduction of Algorithm 6: per row, the best
// (score, word) over the P split lists of length 1, in the strict order
// higher score, then lower word.  One wave per row: each lane scans the
// splits lane, lane + 64, ..., then a wave-wide arg-best.  Empty list slots
// hold scores below every real one, and the split holding the row's maximum
// always lists it.
__global__ __launch_bounds__(256) void k2_argmax(const int2* __restrict__ lists, int P, int N,
                                                 int32_t* __restrict__ tok, float* __restrict__ val) {
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= N) return;  // whole waves leave together
  float bv = -INFINITY;
  int bi = INT_MAX;
  for (int p = lane; p < P; p += 64) {
    const int2 e = lists[(size_t)p * N + r];
    const float v = __int_as_float(e.x);
    if (better(v, e.y, bv, bi)) {
      bv = v;
      bi = e.y;
    }
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    const float ov = __shfl_xor(bv, m, 64);
    const int oi = __shfl_xor(bi, m, 64);
    if (better(ov, oi, bv, bi)) {
      bv = ov;
      bi = oi;
    }
  }
  if (lane == 0) {
    tok[r] = bi;
    val[r] = bv;
  }
}

hipError_t launch_k2_argmax(const int2* lists, int P, int N, int32_t* tok, float* val, hipStream_t st) {
  if (N <= 0) return hipSuccess;
  k2_argmax<<<dim3((N + 3) / 4), dim3(256), 0, st>>>(lists, P, N, tok, val);
  return hipGetLastError();
}

hipError_t launch_k2(const K2Args& a, hipStream_t st) {
  if (a.P > 64 * K2_LPL || a.k > 16) return hipErrorInvalidValue;
  k2_merge<<<dim3(a.S), dim3(256), 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace kb
