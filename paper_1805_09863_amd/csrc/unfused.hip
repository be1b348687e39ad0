// The unfused baseline of the output layer, for the fused-versus-unfused
// comparison of the paper's Section 3 (time per step: multiplication, add
// bias, softmax, k-best extraction).  Every stage is its own kernel and the
// N x V scores live in memory between them:
//
//   mode 0, Algorithm 3 as written: p = W h (stored) -> AddBias -> Softmax
//     (three passes: max, sum, normalise) -> Find-Best extended to the k
//     best of every row -> beam merge;
//   mode 1, Algorithm 4 as the paper runs it: p = W h (stored) -> one fused
//     pass per row (bias, online max/sum, k best) -> beam merge.
//
// The projection is the 256 x 256 MFMA kernel with a store epilogue; the beam
// merge is K2 with a single "split" per row.  The row kernels use one
// 256-thread workgroup per row.
#include "kb_launch.hpp"

namespace kb {

namespace {

constexpr int UF_T = 256;

__device__ __forceinline__ float uf_wave_max(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, __shfl_xor(v, m, 64));
  return v;
}
__device__ __forceinline__ float uf_wave_sum(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
  return v;
}

// workgroup-wide max / sum (4 waves), result in every thread
__device__ float block_max(float v, float* red) {
  v = uf_wave_max(v);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  return fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
}
__device__ float block_sum(float v, float* red) {
  v = uf_wave_sum(v);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  return (red[0] + red[1]) + (red[2] + red[3]);
}

// Sorted (descending, then lower word) list of the KC best in registers; the
// first KC - k slots are +inf sentinels, so the k-th best is slot KC - 1.
template <int KC>
__device__ __forceinline__ void ulist_init(float (&v)[KC], int (&w)[KC], int k) {
#pragma unroll
  for (int j = 0; j < KC; ++j) {
    v[j] = j < KC - k ? INFINITY : -INFINITY;
    w[j] = j < KC - k ? INT_MIN : INT_MAX;
  }
}
template <int KC>
__device__ __forceinline__ void ulist_insert(float (&v)[KC], int (&w)[KC], float x, int i) {
  if (!better(x, i, v[KC - 1], w[KC - 1])) return;
#pragma unroll
  for (int j = 0; j < KC; ++j) {
    const bool bt = better(x, i, v[j], w[j]);
    const float tv = v[j];
    const int tw = w[j];
    v[j] = bt ? x : tv;
    w[j] = bt ? i : tw;
    x = bt ? tv : x;
    i = bt ? tw : i;
  }
}

// Merge the 256 threads' lists (their k real entries) into thread 0's:
// pairwise two-pointer merges in LDS, 8 rounds.
template <int KC>
__device__ void block_merge(float (&v)[KC], int (&w)[KC], int k, float* sv, int* sw) {
  const int t = threadIdx.x;
#pragma unroll
  for (int j = 0; j < KC; ++j)
    if (j >= KC - k) {
      sv[t * 16 + (j - (KC - k))] = v[j];
      sw[t * 16 + (j - (KC - k))] = w[j];
    }
  __syncthreads();
  for (int step = 1; step < UF_T; step <<= 1) {
    if ((t & (2 * step - 1)) == 0) {
      const int o = t + step;
      float mv[KC];
      int mw[KC];
      int a = 0, c = 0;
#pragma unroll
      for (int j = 0; j < KC; ++j) {
        if (j < k) {  // (a, c < k: each list holds k entries)
          const bool ta = better(sv[t * 16 + a], sw[t * 16 + a], sv[o * 16 + c], sw[o * 16 + c]);
          mv[j] = ta ? sv[t * 16 + a] : sv[o * 16 + c];
          mw[j] = ta ? sw[t * 16 + a] : sw[o * 16 + c];
          a += ta ? 1 : 0;
          c += ta ? 0 : 1;
        }
      }
#pragma unroll
      for (int j = 0; j < KC; ++j)
        if (j < k) {
          sv[t * 16 + j] = mv[j];
          sw[t * 16 + j] = mw[j];
        }
    }
    __syncthreads();
  }
}

__global__ __launch_bounds__(UF_T) void uf_add_bias(float4* __restrict__ x, const float4* __restrict__ b, int N,
                                                   int V4) {
  const long long total = (long long)N * V4;
  for (long long i = (long long)blockIdx.x * UF_T + threadIdx.x; i < total; i += (long long)gridDim.x * UF_T) {
    float4 v = x[i];
    const float4 c = b[i % V4];
    v.x += c.x;
    v.y += c.y;
    v.z += c.z;
    v.w += c.w;
    x[i] = v;
  }
}

// Algorithm 3 Softmax: three passes over the row (max; sum of exp(x - max);
// normalise in place).  row_lse (nullable) receives max + ln(sum).
__global__ __launch_bounds__(UF_T) void uf_softmax3(float* __restrict__ x, int V, float* __restrict__ row_lse) {
  __shared__ float red[8];
  float4* r = reinterpret_cast<float4*>(x + (size_t)blockIdx.x * V);
  const int V4 = V / 4;
  float m = -INFINITY;
  for (int i = threadIdx.x; i < V4; i += UF_T) {
    const float4 v = r[i];
    m = fmaxf(fmaxf(m, fmaxf(v.x, v.y)), fmaxf(v.z, v.w));
  }
  m = block_max(m, red);
  float s = 0.f;
  for (int i = threadIdx.x; i < V4; i += UF_T) {
    const float4 v = r[i];
    s += (expf(v.x - m) + expf(v.y - m)) + (expf(v.z - m) + expf(v.w - m));
  }
  s = block_sum(s, red + 4);
  if (row_lse && threadIdx.x == 0) row_lse[blockIdx.x] = m + logf(s);
  const float inv = 1.f / s;
  for (int i = threadIdx.x; i < V4; i += UF_T) {
    float4 v = r[i];
    v.x = expf(v.x - m) * inv;
    v.y = expf(v.y - m) * inv;
    v.z = expf(v.z - m) * inv;
    v.w = expf(v.w - m) * inv;
    r[i] = v;
  }
}

// Algorithm 3 Find-Best for the k best of every row of probabilities p.
// Output in the partial format of the fused kernel with one split: scores
// log p (statistics (0, 1), so that the merge's log-sum-exp is 0).
template <int KC>
__global__ __launch_bounds__(UF_T) void uf_kbest_rows(const float* __restrict__ p, int V, int k,
                                                      float2* __restrict__ stats, int2* __restrict__ lists) {
  __shared__ float sv[UF_T * 16];
  __shared__ int sw[UF_T * 16];
  const float4* r = reinterpret_cast<const float4*>(p + (size_t)blockIdx.x * V);
  float v[KC];
  int w[KC];
  ulist_init<KC>(v, w, k);
  for (int i = threadIdx.x; i < V / 4; i += UF_T) {
    const float4 q = r[i];
    ulist_insert<KC>(v, w, q.x, 4 * i);
    ulist_insert<KC>(v, w, q.y, 4 * i + 1);
    ulist_insert<KC>(v, w, q.z, 4 * i + 2);
    ulist_insert<KC>(v, w, q.w, 4 * i + 3);
  }
  block_merge<KC>(v, w, k, sv, sw);
  if (threadIdx.x < k) {
    const size_t row = blockIdx.x;
    lists[row * k + threadIdx.x] = make_int2(__float_as_int(logf(sv[threadIdx.x])), sw[threadIdx.x]);
  }
  if (threadIdx.x == 0) stats[blockIdx.x] = make_float2(0.f, 1.f);
}

// Algorithm 4 as a separate pass over stored scores: bias, running max and
// sum (one rescale per thread-local maximum change) and the k best, in one
// read of the row.
template <int KC>
__global__ __launch_bounds__(UF_T) void uf_fused_rows(const float* __restrict__ x, const float* __restrict__ b,
                                                      int V, int k, float2* __restrict__ stats,
                                                      int2* __restrict__ lists) {
  __shared__ float sv[UF_T * 16];
  __shared__ int sw[UF_T * 16];
  __shared__ float red[8];
  const float4* r = reinterpret_cast<const float4*>(x + (size_t)blockIdx.x * V);
  const float4* b4 = reinterpret_cast<const float4*>(b);
  float v[KC];
  int w[KC];
  ulist_init<KC>(v, w, k);
  float m = -INFINITY, s = 0.f;
  for (int i = threadIdx.x; i < V / 4; i += UF_T) {
    float4 q = r[i];
    const float4 c = b4[i];
    q.x += c.x;
    q.y += c.y;
    q.z += c.z;
    q.w += c.w;
    const float mx = fmaxf(fmaxf(q.x, q.y), fmaxf(q.z, q.w));
    if (mx > m) {
      s *= expf(m - mx);
      m = mx;
    }
    s += (expf(q.x - m) + expf(q.y - m)) + (expf(q.z - m) + expf(q.w - m));
    ulist_insert<KC>(v, w, q.x, 4 * i);
    ulist_insert<KC>(v, w, q.y, 4 * i + 1);
    ulist_insert<KC>(v, w, q.z, 4 * i + 2);
    ulist_insert<KC>(v, w, q.w, 4 * i + 3);
  }
  // combine the threads' (max, sum) with the rescaling identity
  const float M = block_max(m, red);
  const float S = block_sum(m == -INFINITY ? 0.f : s * expf(m - M), red + 4);
  block_merge<KC>(v, w, k, sv, sw);
  if (threadIdx.x < k) {
    const size_t row = blockIdx.x;
    lists[row * k + threadIdx.x] = make_int2(__float_as_int(sv[threadIdx.x]), sw[threadIdx.x]);
  }
  if (threadIdx.x == 0) stats[blockIdx.x] = make_float2(M, S);
}

}  // namespace

hipError_t launch_uf_add_bias(float* x, const float* b, int N, int V, hipStream_t st) {
  const long long total = (long long)N * (V / 4);
  const long long want = (total + UF_T - 1) / UF_T;
  const int blocks = (int)(want < 8192 ? want : 8192);
  uf_add_bias<<<dim3(blocks > 0 ? blocks : 1), dim3(UF_T), 0, st>>>(
      reinterpret_cast<float4*>(x), reinterpret_cast<const float4*>(b), N, V / 4);
  return hipGetLastError();
}

hipError_t launch_uf_softmax3(float* x, int N, int V, float* row_lse, hipStream_t st) {
  uf_softmax3<<<dim3(N), dim3(UF_T), 0, st>>>(x, V, row_lse);
  return hipGetLastError();
}

hipError_t launch_uf_kbest_rows(const float* p, int N, int V, int k, float2* stats, int2* lists, hipStream_t st) {
  const dim3 g(N), t(UF_T);
  if (k <= 4) uf_kbest_rows<4><<<g, t, 0, st>>>(p, V, k, stats, lists);
  else if (k <= 8) uf_kbest_rows<8><<<g, t, 0, st>>>(p, V, k, stats, lists);
  else if (k <= 12) uf_kbest_rows<12><<<g, t, 0, st>>>(p, V, k, stats, lists);
  else uf_kbest_rows<16><<<g, t, 0, st>>>(p, V, k, stats, lists);
  return hipGetLastError();
}

hipError_t launch_uf_fused_rows(const float* x, const float* b, int N, int V, int k, float2* stats, int2* lists,
                                hipStream_t st) {
  const dim3 g(N), t(UF_T);
  if (k <= 4) uf_fused_rows<4><<<g, t, 0, st>>>(x, b, V, k, stats, lists);
  else if (k <= 8) uf_fused_rows<8><<<g, t, 0, st>>>(x, b, V, k, stats, lists);
  else if (k <= 12) uf_fused_rows<12><<<g, t, 0, st>>>(x, b, V, k, stats, lists);
  else uf_fused_rows<16><<<g, t, 0, st>>>(x, b, V, k, stats, lists);
  return hipGetLastError();
}

}  // namespace kb
