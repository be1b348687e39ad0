// K1, few-row variant: the fused output-layer projection when a step has at
// most FEW_ROWS live rows (a few sentences left in the batch, or one short
// beam).  Such a step is bound by reading W once (a few flops per weight), so
// this kernel does not use the matrix cores: it streams W with 16-byte loads
// into plain FMAs (float32) or two-state dot products (bf16), with every
// row's state h held in LDS, and turns each chunk of words straight into the
// row's softmax statistics and k best.
//
// Workgroup j takes the word chunks j*tps .. (j+1)*tps-1 (a "split" in the
// terms of the merge kernel).  Its first W loads are issued before the
// states and the split's bias are copied to LDS, so the three arrive in one
// memory round trip.  Per chunk of CW words, thread (s, g) (16 state
// slices x 16 word groups) accumulates the scores of WPT consecutive words
// over its slice of the states for every row; the 16 slices are summed
// through LDS, the bias is added, and one wave per row folds the chunk into
// the row's running (max, sum of exp) -- Algorithm 4's rescaling, once per
// chunk -- and its sorted k-list (k rounds of a wave-wide maximum over
// 64-bit keys whose order is the strict one: higher score, then lower word;
// branch-free, so a round is a short chain of DPP and scalar maxima).  The
// split's statistics and list
// go to the same partial arrays the MFMA kernels fill, for the same merge.
// No shared thresholds are used, so nothing needs resetting per call.
#include <type_traits>

#include "kb_launch.hpp"
#include "wave_keys.hpp"

namespace kb {

namespace {

constexpr int kFewSlices = 16;  // state slices per chunk
constexpr int kFewGroups = 16;  // word groups per chunk

template <int CTRL>
__device__ __forceinline__ float few_dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
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

// NR: the step's row count rounded up to 1, 2, 4 or 8.  The row loops are
// unrolled over NR without early exits (rows N .. NR-1 repeat row N-1's state;
// their sums are never read), which keeps the kernel's code a few KB: one
// version for every row count with early exits made the float32 kernel
// 78 KB, more than the instruction cache, and each launch ran it cold.
template <class T, int NR>
__global__ __launch_bounds__(256) void k1_few(K1Args a) {
  using G = FewGeom<T>;
  constexpr int WPT = G::WPT, CW = G::CW, KSTEP = G::KSTEP, GS = G::GS;
  constexpr int QW = (NR + 3) / 4;  // rows per wave in the row epilogue
  extern __shared__ __align__(16) unsigned char few_lds[];
  float* part = reinterpret_cast<float*>(few_lds);                   // [16 slices][NR][CW]
  float* bl = part + kFewSlices * NR * CW;                          // [tps * CW] the split's bias
  T* hl = reinterpret_cast<T*>(bl + (size_t)a.tps * CW);            // [N][H] states

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = tid & (kFewGroups - 1), sl = tid >> 4;
  const int N = a.N, H = a.H, V = a.V, k = a.k;
  const int split = blockIdx.x;
  const int c0 = split * a.tps, c1 = min(c0 + a.tps, a.n_vtiles);

  // this thread's slice of the states: steps [ks0, ks1) of KSTEP states each,
  // slices a multiple of 4 steps long (16-byte reads of the states in LDS)
  const int nsteps = H / KSTEP;
  const int per = (((nsteps + kFewSlices - 1) / kFewSlices) + 3) & ~3;
  const int ks0 = min(sl * per, nsteps), ks1 = min(ks0 + per, nsteps);
  const int ngr = (per + GS - 1) / GS;           // load groups per chunk (the same for every slice)
  const int total = (c1 - c0) * ngr;

  // running statistics and k-list of the rows this wave owns (rows wave, wave + 4):
  // lane r < k holds the key of the r-th best (score, word) of the split so far
  float st_m[QW], st_s[QW];
  uint64_t lk[QW];
#pragma unroll
  for (int q = 0; q < QW; ++q) {
    st_m[q] = kStatInit;
    st_s[q] = 0.f;
    lk[q] = kEmptyKey;
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
      part[n * CW + w] = word < V ? x + bl[word - c0 * CW] : -INFINITY;  // slice 0's storage, rows [0, N)
    }
    __syncthreads();
    uint64_t ck[QW][G::PER_LANE];  // the chunk's candidates of each row (empty keys where none)
    bool need = false;
#pragma unroll
    for (int q = 0; q < QW; ++q) {
      const int n = wave + 4 * q;
#pragma unroll
      for (int j = 0; j < G::PER_LANE; ++j) ck[q][j] = kEmptyKey;
      if (n >= N) continue;
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
      // k-list: left as it is when no word of the chunk can enter (all below the k-th best)
      const float kth = key_score(readlane64(lk[q], k - 1));
      if (cm < kth) continue;
      need = true;
#pragma unroll
      for (int j = 0; j < G::PER_LANE; ++j) ck[q][j] = key_of(x[j], xw[j]);  // masked words: the empty key
    }
    if (need) {
      // k rounds, the wave's rows side by side: the wave-wide largest key
      // among the list and the chunk's candidates goes to lane r, and its
      // holder replaces it by the empty key (real words are distinct; empty
      // keys are all alike, and taking one leaves the others as they are)
      uint64_t nk[QW];
#pragma unroll
      for (int q = 0; q < QW; ++q) nk[q] = kEmptyKey;
      for (int r = 0; r < k; ++r) {
#pragma unroll
        for (int q = 0; q < QW; ++q) {
          uint64_t best = lk[q];
#pragma unroll
          for (int j = 0; j < G::PER_LANE; ++j) best = ck[q][j] > best ? ck[q][j] : best;
          const uint64_t win = wave_max64(best);
          nk[q] = lane == r ? win : nk[q];
          lk[q] = lk[q] == win ? kEmptyKey : lk[q];
#pragma unroll
          for (int j = 0; j < G::PER_LANE; ++j) ck[q][j] = ck[q][j] == win ? kEmptyKey : ck[q][j];
        }
      }
#pragma unroll
      for (int q = 0; q < QW; ++q) lk[q] = lane < k ? nk[q] : kEmptyKey;
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
        hv[n] = *reinterpret_cast<const u32x4v*>(hl + (size_t)min(n, N - 1) * H + (size_t)(st0 + u4) * KSTEP);
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
            const uint32_t hp = hv[n][u - u4];
#pragma unroll
            for (int j = 0; j < WPT; ++j)
              acc[n][j] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2v, wp[j]),
                                                          __builtin_bit_cast(bf16x2v, hp), acc[n][j], false);
          }
        } else {
#pragma unroll
          for (int n = 0; n < NR; ++n) {
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
  // the first two load groups, then every row's state (16-byte copies;
  // N * H * sizeof(T) is a multiple of 16) and the split's bias (masked past V)
  // into LDS: the copies' waits cover the W loads issued before them
  issue(B0{}, 0);
  issue(B1{}, 1);
  {
    const int wb0 = c0 * CW, nw = (c1 - c0) * CW;
    // Copies without branches (a branch around a load or store drew a wait for
    // every load in flight, the W groups' included): indexes are clamped to the
    // last element, and threads past the end copy that element again.
    const int j0 = min(tid, nw - 1);
    const float b0 = a.b[min(wb0 + j0, V - 1)];
    const u32x4v* src = reinterpret_cast<const u32x4v*>(a.h);
    u32x4v* dst = reinterpret_cast<u32x4v*>(hl);
    const int n16 = (int)((size_t)N * H * sizeof(T) / 16);  // >= 1
    for (int i0 = 0; i0 < n16; i0 += 1024) {  // four loads in flight per thread before the LDS writes
      u32x4v t4[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) t4[u] = src[min(i0 + u * 256 + tid, n16 - 1)];
#pragma unroll
      for (int u = 0; u < 4; ++u) dst[min(i0 + u * 256 + tid, n16 - 1)] = t4[u];
    }
    bl[j0] = wb0 + j0 < V ? b0 : 0.f;
    for (int i = tid + 256; i < nw; i += 256) bl[i] = wb0 + i < V ? a.b[wb0 + i] : 0.f;
  }
  __syncthreads();  // the states and the bias in LDS
  for (int gi = 0; gi < total; gi += 2) {
    compute(B0{}, gi);
    if (gi + 1 >= total) break;
    issue(B0{}, gi + 2);
    compute(B1{}, gi + 1);
    issue(B1{}, gi + 3);
  }

  // this split's partials: (max, sum) and the sorted k-list of every row
#pragma unroll
  for (int q = 0; q < QW; ++q) {
    const int n = wave + 4 * q;
    if (n >= N) break;
    const size_t row = (size_t)split * N + n;
    if (lane == 0) a.stats[row] = make_float2(st_m[q], st_s[q]);
    if (lane < k) a.lists[row * k + lane] = make_int2(__float_as_int(key_score(lk[q])), key_index(lk[q]));
  }
}

template <class T>
size_t few_lds_bytes(int N, int H, int tps) {
  return (size_t)kFewSlices * FEW_ROWS * FewGeom<T>::CW * 4 + (size_t)tps * FewGeom<T>::CW * 4 +
         (size_t)N * H * sizeof(T);
}

template <class T, int NR>
hipError_t launch_few_nr(dim3 grid, const K1Args& a, hipStream_t st) {
  const size_t lds = few_lds_bytes<T>(a.N, a.H, a.tps);
  static bool attr_set = false;  // the kernel's LDS ceiling, raised once per process
  if (!attr_set) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k1_few<T, NR>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  k1_few<T, NR><<<grid, dim3(256), lds, st>>>(a);
  return hipGetLastError();
}

template <class T>
hipError_t launch_few(dim3 grid, const K1Args& a, hipStream_t st) {
  if (a.N < 1 || a.N > FEW_ROWS) return hipErrorInvalidValue;
  if (a.N == 1) return launch_few_nr<T, 1>(grid, a, st);
  if (a.N == 2) return launch_few_nr<T, 2>(grid, a, st);
  if (a.N <= 4) return launch_few_nr<T, 4>(grid, a, st);
  return launch_few_nr<T, 8>(grid, a, st);
}

}  // namespace

int few_chunk_words(int bf16) { return bf16 ? FewGeom<__bf16>::CW : FewGeom<float>::CW; }

size_t few_lds_needed(int bf16, int N, int H, int tps) {
  return bf16 ? few_lds_bytes<__bf16>(N, H, tps) : few_lds_bytes<float>(N, H, tps);
}

hipError_t launch_k1_few(int bf16, dim3 grid, const K1Args& a, hipStream_t st) {
  return bf16 ? launch_few<__bf16>(grid, a, st) : launch_few<float>(grid, a, st);
}

}  // namespace kb
