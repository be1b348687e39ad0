// K1, few-row variant: the fused output-layer projection when a step has at
// most FEW_ROWS live rows (a few sentences left in the batch, or one short
// beam).  Such a step is bound by reading W once (a few flops per weight), so
// this kernel does not use the matrix cores: it streams W with 16-byte loads
// into plain FMAs (float32) or two-state dot products (bf16), with every
// row's state h held in LDS, and turns each chunk of words straight into the
// row's softmax statistics and k best.
//
// Workgroup j takes the word chunks j*tps .. (j+1)*tps-1 (a "split" in the
// terms of the merge kernel).  Per chunk of CW words, thread (s, g) (16 state
// slices x 16 word groups) accumulates the scores of WPT consecutive words
// over its slice of the states for every row; the 16 slices are summed
// through LDS, the bias is added, and one wave per row folds the chunk into
// the row's running (max, sum of exp) -- Algorithm 4's rescaling, once per
// chunk -- and its sorted k-list (k rounds of a wave-wide arg-best, strict
// order: higher score, then lower word).  The split's statistics and list
// go to the same partial arrays the MFMA kernels fill, for the same merge.
// No shared thresholds are used, so nothing needs resetting per call.
#include <type_traits>

#include "kb_launch.hpp"

namespace kb {

namespace {

constexpr int kFewSlices = 16;  // state slices per chunk
constexpr int kFewGroups = 16;  // word groups per chunk

template <int CTRL>
__device__ __forceinline__ float few_dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
template <int CTRL>
__device__ __forceinline__ int few_dpp_i(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false);
}
constexpr int kXor1 = 0xB1, kXor2 = 0x4E, kHalfMirror = 0x141, kMirror = 0x140;
__device__ __forceinline__ float rl_f(float v, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}
__device__ __forceinline__ float few_wave_max(float v) {
  v = fmaxf(v, few_dpp_f<kXor1>(v));
  v = fmaxf(v, few_dpp_f<kXor2>(v));
  v = fmaxf(v, few_dpp_f<kHalfMirror>(v));
  v = fmaxf(v, few_dpp_f<kMirror>(v));
  return fmaxf(fmaxf(rl_f(v, 0), rl_f(v, 16)), fmaxf(rl_f(v, 32), rl_f(v, 48)));
}
__device__ __forceinline__ float few_wave_sum(float v) {
  v += few_dpp_f<kXor1>(v);
  v += few_dpp_f<kXor2>(v);
  v += few_dpp_f<kHalfMirror>(v);
  v += few_dpp_f<kMirror>(v);
  return (rl_f(v, 0) + rl_f(v, 16)) + (rl_f(v, 32) + rl_f(v, 48));
}
template <int CTRL>
__device__ __forceinline__ void few_argbest_step(float& v, int& i) {
  const float ov = few_dpp_f<CTRL>(v);
  const int oi = few_dpp_i<CTRL>(i);
  if (better(ov, oi, v, i)) {
    v = ov;
    i = oi;
  }
}
// the best (score, word) of the wave under better(); every lane gets it
__device__ __forceinline__ void few_wave_argbest(float& v, int& i) {
  few_argbest_step<kXor1>(v, i);
  few_argbest_step<kXor2>(v, i);
  few_argbest_step<kHalfMirror>(v, i);
  few_argbest_step<kMirror>(v, i);
  float bv = rl_f(v, 0);
  int bi = __builtin_amdgcn_readlane(i, 0);
#pragma unroll
  for (int l = 16; l < 64; l += 16) {
    const float ov = rl_f(v, l);
    const int oi = __builtin_amdgcn_readlane(i, l);
    if (better(ov, oi, bv, bi)) {
      bv = ov;
      bi = oi;
    }
  }
  v = bv;
  i = bi;
}

typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2v __attribute__((ext_vector_type(2)));

template <class T>
struct FewGeom {
  static constexpr bool BF16 = sizeof(T) == 2;
  static constexpr int WPT = 16 / sizeof(T);        // words per 16-byte load
  static constexpr int CW = kFewGroups * WPT;       // words per chunk
  static constexpr int PER_LANE = CW / 64;          // chunk words per lane in the row epilogue
  static constexpr int KSTEP = BF16 ? 2 : 1;        // states per step (a bf16 pair)
  static constexpr int GS = BF16 ? 8 : 16;          // steps per load group (16 loads of 16 bytes)
};

template <class T>
__global__ __launch_bounds__(256) void k1_few(K1Args a) {
  using G = FewGeom<T>;
  constexpr int WPT = G::WPT, CW = G::CW, NR = FEW_ROWS, KSTEP = G::KSTEP, GS = G::GS;
  extern __shared__ __align__(16) unsigned char few_lds[];
  float* part = reinterpret_cast<float*>(few_lds);                  // [16 slices][NR][CW]
  T* hl = reinterpret_cast<T*>(few_lds + kFewSlices * NR * CW * 4);  // [N][H] states

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = tid & (kFewGroups - 1), sl = tid >> 4;
  const int N = a.N, H = a.H, V = a.V, k = a.k;
  const int split = blockIdx.x;
  const int c0 = split * a.tps, c1 = min(c0 + a.tps, a.n_vtiles);

  // every row's state into LDS (16-byte copies; N * H * sizeof(T) is a multiple of 16)
  {
    const u32x4v* src = reinterpret_cast<const u32x4v*>(a.h);
    u32x4v* dst = reinterpret_cast<u32x4v*>(hl);
    const int n16 = (int)((size_t)N * H * sizeof(T) / 16);
    for (int i = tid; i < n16; i += 256) dst[i] = src[i];
  }

  // this thread's slice of the states: steps [ks0, ks1) of KSTEP states each,
  // slices a multiple of 4 steps long (16-byte reads of the states in LDS)
  const int nsteps = H / KSTEP;
  const int per = (((nsteps + kFewSlices - 1) / kFewSlices) + 3) & ~3;
  const int ks0 = min(sl * per, nsteps), ks1 = min(ks0 + per, nsteps);
  const int ngr = (per + GS - 1) / GS;           // load groups per chunk (the same for every slice)
  const int total = (c1 - c0) * ngr;

  // running statistics and k-list of the rows this wave owns (rows wave, wave + 4):
  // lane r < k holds the r-th best (score, word) of the split so far
  float st_m[NR / 4], st_s[NR / 4], lv[NR / 4];
  int li[NR / 4];
#pragma unroll
  for (int q = 0; q < NR / 4; ++q) {
    st_m[q] = kStatInit;
    st_s[q] = 0.f;
    lv[q] = -INFINITY;
    li[q] = INT_MAX;
  }

  const size_t rowb = (size_t)V * sizeof(T);
  // W of load group gi (chunk c0 + gi / ngr, steps of group gi % ngr of this
  // thread's slice): two groups in flight, the next issued before the current is used
  u32x4v wb[2][GS][KSTEP];
  auto issue = [&](auto bc, int gi) __attribute__((always_inline)) {
    constexpr int B = decltype(bc)::value;
    if (gi >= total) return;
    const int c = c0 + gi / ngr, q = gi - (gi / ngr) * ngr;
    const int st0 = ks0 + q * GS;
    if (st0 >= ks1) return;                      // nothing of this group in the slice
    const int wv0 = min(c * CW + g * WPT, V - WPT);  // clamped in the ragged last chunk (masked later)
    const char* wbase = reinterpret_cast<const char*>(a.W) + (size_t)wv0 * sizeof(T);
#pragma unroll
    for (int u = 0; u < GS; ++u) {
      const int s = min(st0 + u, ks1 - 1);       // clamped: steps past the slice are loaded, not used
#pragma unroll
      for (int e = 0; e < KSTEP; ++e)
        wb[B][u][e] = *reinterpret_cast<const u32x4v*>(wbase + (size_t)(s * KSTEP + e) * rowb);
    }
  };

  float acc[NR][WPT];
  // one chunk's scores are complete: sum the slices, add the bias, and fold
  // them into each row's statistics and k-list (one wave per row)
  auto finish_chunk = [&](int c) __attribute__((always_inline)) {
    const int v0 = c * CW;
#pragma unroll
    for (int n = 0; n < NR; ++n) {
      if (n >= N) break;
#pragma unroll
      for (int j = 0; j < WPT; j += 4)
        *reinterpret_cast<float4*>(&part[(sl * NR + n) * CW + g * WPT + j]) =
            make_float4(acc[n][j], acc[n][j + 1], acc[n][j + 2], acc[n][j + 3]);
    }
    __syncthreads();
    for (int i = tid; i < N * CW; i += 256) {
      const int n = i / CW, w = i - n * CW;
      float x = 0.f;
#pragma unroll
      for (int s = 0; s < kFewSlices; ++s) x += part[(s * NR + n) * CW + w];
      const int word = v0 + w;
      part[n * CW + w] = word < V ? x + a.b[word] : -INFINITY;  // slice 0's storage, rows [0, N)
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < NR / 4; ++q) {
      const int n = wave + 4 * q;
      if (n >= N) break;
      float x[G::PER_LANE];
      int xw[G::PER_LANE];
#pragma unroll
      for (int j = 0; j < G::PER_LANE; ++j) {
        x[j] = part[n * CW + lane + 64 * j];
        xw[j] = v0 + lane + 64 * j < V ? v0 + lane + 64 * j : INT_MAX;  // masked words: empty entries
      }
      float cm = x[0];
#pragma unroll
      for (int j = 1; j < G::PER_LANE; ++j) cm = fmaxf(cm, x[j]);
      cm = few_wave_max(cm);
      // statistics (a chunk of only masked words leaves them unchanged)
      const float mnew = fmaxf(st_m[q], cm);
      float se = 0.f;
#pragma unroll
      for (int j = 0; j < G::PER_LANE; ++j) se += exp2_fast((x[j] - mnew) * kL2E);
      se = few_wave_sum(se);
      st_s[q] = st_s[q] * exp2_fast((st_m[q] - mnew) * kL2E) + se;
      st_m[q] = mnew;
      // k-list: skipped when no word of the chunk can enter (all below the k-th best)
      const float kth = rl_f(lv[q], k - 1);
      if (cm < kth) continue;
      bool taken[G::PER_LANE];
#pragma unroll
      for (int j = 0; j < G::PER_LANE; ++j) taken[j] = false;
      bool ltaken = lane >= k;
      float nv = -INFINITY;
      int ni = INT_MAX;
      for (int r = 0; r < k; ++r) {
        float bv = ltaken ? -INFINITY : lv[q];
        int bi = ltaken ? INT_MAX : li[q];
#pragma unroll
        for (int j = 0; j < G::PER_LANE; ++j)
          if (!taken[j] && better(x[j], xw[j], bv, bi)) {
            bv = x[j];
            bi = xw[j];
          }
        float wv = bv;
        int wi = bi;
        few_wave_argbest(wv, wi);
        if (lane == r) {
          nv = wv;
          ni = wi;
        }
        // the holder of the winner gives it up (real words are distinct)
        if (!ltaken && li[q] == wi && lv[q] == wv) ltaken = true;
#pragma unroll
        for (int j = 0; j < G::PER_LANE; ++j)
          if (!taken[j] && xw[j] == wi && x[j] == wv) taken[j] = true;
      }
      lv[q] = lane < k ? nv : -INFINITY;
      li[q] = lane < k ? ni : INT_MAX;
    }
    __syncthreads();  // the chunk's scores are read before the next chunk's slices land
  };

  auto compute = [&](auto bc, int gi) __attribute__((always_inline)) {
    constexpr int B = decltype(bc)::value;
    const int c = c0 + gi / ngr, q = gi - (gi / ngr) * ngr;
    if (q == 0) {
#pragma unroll
      for (int n = 0; n < NR; ++n)
#pragma unroll
        for (int j = 0; j < WPT; ++j) acc[n][j] = 0.f;
    }
    const int st0 = ks0 + q * GS;
#pragma unroll
    for (int u4 = 0; u4 < GS; u4 += 4) {
      if (st0 + u4 >= ks1) break;                // slices end on a multiple of 4 steps, or at H
      // states of steps st0 + u4 .. + 3 of every row: one 16-byte LDS read per row
      u32x4v hv[NR];
#pragma unroll
      for (int n = 0; n < NR; ++n)
        if (n < N) hv[n] = *reinterpret_cast<const u32x4v*>(hl + (size_t)n * H + (size_t)(st0 + u4) * KSTEP);
#pragma unroll
      for (int u = u4; u < u4 + 4; ++u) {
        if (st0 + u >= ks1) break;
        if constexpr (G::BF16) {
          // (state 2s, state 2s + 1) pairs of each word, for the two-state dot product
          uint32_t wp[WPT];
#pragma unroll
          for (int d = 0; d < 4; ++d) {
            wp[2 * d] = __builtin_amdgcn_perm(wb[B][u][1][d], wb[B][u][0][d], 0x05040100u);
            wp[2 * d + 1] = __builtin_amdgcn_perm(wb[B][u][1][d], wb[B][u][0][d], 0x07060302u);
          }
#pragma unroll
          for (int n = 0; n < NR; ++n) {
            if (n >= N) break;
            const uint32_t hp = hv[n][u - u4];
#pragma unroll
            for (int j = 0; j < WPT; ++j)
              acc[n][j] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2v, wp[j]),
                                                          __builtin_bit_cast(bf16x2v, hp), acc[n][j], false);
          }
        } else {
#pragma unroll
          for (int n = 0; n < NR; ++n) {
            if (n >= N) break;
            const float hs = __uint_as_float(hv[n][u - u4]);
#pragma unroll
            for (int j = 0; j < WPT; ++j) acc[n][j] = fmaf(__uint_as_float(wb[B][u][0][j]), hs, acc[n][j]);
          }
        }
      }
    }
    if (q == ngr - 1) finish_chunk(c);
  };

  using B0 = std::integral_constant<int, 0>;
  using B1 = std::integral_constant<int, 1>;
  issue(B0{}, 0);
  __syncthreads();  // the states in LDS
  for (int gi = 0; gi < total; gi += 2) {
    issue(B1{}, gi + 1);
    compute(B0{}, gi);
    if (gi + 1 >= total) break;
    issue(B0{}, gi + 2);
    compute(B1{}, gi + 1);
  }

  // this split's partials: (max, sum) and the sorted k-list of every row
#pragma unroll
  for (int q = 0; q < NR / 4; ++q) {
    const int n = wave + 4 * q;
    if (n >= N) break;
    const size_t row = (size_t)split * N + n;
    if (lane == 0) a.stats[row] = make_float2(st_m[q], st_s[q]);
    if (lane < k) a.lists[row * k + lane] = make_int2(__float_as_int(lv[q]), li[q]);
  }
}

template <class T>
size_t few_lds_bytes(int N, int H) {
  return (size_t)kFewSlices * FEW_ROWS * FewGeom<T>::CW * 4 + (size_t)N * H * sizeof(T);
}

template <class T>
hipError_t launch_few(dim3 grid, const K1Args& a, hipStream_t st) {
  const size_t lds = few_lds_bytes<T>(a.N, a.H);
  static bool attr_set = false;  // the kernel's LDS ceiling, raised once per process
  if (!attr_set) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k1_few<T>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  k1_few<T><<<grid, dim3(256), lds, st>>>(a);
  return hipGetLastError();
}

}  // namespace

int few_chunk_words(int bf16) { return bf16 ? FewGeom<__bf16>::CW : FewGeom<float>::CW; }

size_t few_lds_needed(int bf16, int N, int H) {
  return bf16 ? few_lds_bytes<__bf16>(N, H) : few_lds_bytes<float>(N, H);
}

hipError_t launch_k1_few(int bf16, dim3 grid, const K1Args& a, hipStream_t st) {
  return bf16 ? launch_few<__bf16>(grid, a, st) : launch_few<float>(grid, a, st);
}

}  // namespace kb
