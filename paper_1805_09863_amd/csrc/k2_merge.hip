// K2: merge the vocabulary splits of every row, then the rows of every sentence.
//
// One workgroup per sentence, W waves (one per row of an average sentence,
// W <= 16, and no more than the staged lists fit in LDS); the sentence's rows
// are taken W at a time, one per wave:
//   * the row's P split lists are staged in LDS, eight or sixteen loads in
//     flight per lane, and its P split statistics held in registers;
//   * LSE = M + ln(sum_p s_p * exp(m_p - M)) over the P split partials -- the
//     rescaling identity of Algorithm 4 applied between shards, the reduction
//     step of Algorithm 6 extended from (max, best) to softmax statistics;
//   * the row's best words: rounds of a wave-wide maximum of 64-bit keys
//     (wave_keys.hpp) over the heads of the P sorted split lists (strict
//     total order: higher score, then lower word).  Each lane keeps its lists' heads and the entries
//     after them in registers, so a round reads no LDS on its critical path.
//     The rounds stop once a score (prev + x - LSE) falls below the sentence's
//     k-th best so far: the row's later entries are worse still;
//   * the running k best of the sentence and the chunk's candidates are ranked
//     by (score desc, flat index asc), flat index being
//     (row - first row) * V + word, one thread per candidate, and the first k
//     kept.  Because the score adds a per-row constant to x, a sentence's k
//     best lie in the union of its rows' k best, so nothing outside these
//     candidates can be selected.
#include "kb_launch.hpp"
#include "wave_keys.hpp"

namespace kb {

constexpr int K2_MAXW = 16;                  // waves per workgroup: rows merged at once
constexpr int K2_LPL = 4;                    // split lists per lane: P <= 256
constexpr int K2_LS = 16;                    // LDS slots per staged split list (k <= 16)
constexpr int K2_C = K2_MAXW * 16 + 16 + 2;  // running best + one chunk (+ pad to pairs)
constexpr int kNegInfBits = (int)0xff800000;  // -inf: the score of an empty entry (word INT_MAX)
static_assert(K2_C % 2 == 0, "candidate keys are read in pairs");

// Wave-wide reductions from DPP moves within each row of 16 lanes (quad
// xor 1, quad xor 2, half-row mirror, row mirror), then the four row results
// read out (v_readlane): no LDS permutes on the merge's critical path.
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
constexpr int kDppXor1 = 0xB1, kDppXor2 = 0x4E, kDppHalfMirror = 0x141, kDppMirror = 0x140;
__device__ __forceinline__ float lane_f(float v, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}

__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp_f<kDppXor1>(v));
  v = fmaxf(v, dpp_f<kDppXor2>(v));
  v = fmaxf(v, dpp_f<kDppHalfMirror>(v));
  v = fmaxf(v, dpp_f<kDppMirror>(v));
  return fmaxf(fmaxf(lane_f(v, 0), lane_f(v, 16)), fmaxf(lane_f(v, 32), lane_f(v, 48)));
}
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_f<kDppXor1>(v);
  v += dpp_f<kDppXor2>(v);
  v += dpp_f<kDppHalfMirror>(v);
  v += dpp_f<kDppMirror>(v);
  return (lane_f(v, 0) + lane_f(v, 16)) + (lane_f(v, 32) + lane_f(v, 48));
}
// A candidate of the sentence merge as one 64-bit key (key_of) of its score
// and flat index: a higher score, then a lower flat index, gives the larger key.
__device__ __forceinline__ uint64_t cand_key(float score, int flat) { return key_of(score, flat); }

// NQ: split lists per lane (P <= 64 * NQ); MAXT: the workgroup size it is
// compiled for (1024: up to 16 waves, 128 VGPRs; 512: up to 8, 256 VGPRs,
// which lets a lane keep a whole row's staging loads in flight)
template <int NQ, int MAXT>
__global__ __launch_bounds__(MAXT) void k2_merge(K2Args a) {
  __shared__ __align__(16) uint64_t key[K2_C];  // read two at a time when ranked
  __shared__ int c_t[K2_C];
  __shared__ int c_p[K2_C];
  __shared__ uint64_t n_key[16];
  __shared__ int n_t[16], n_p[16];
  // one list of empty entries, then per wave one row's P lists of K2_LS slots
  extern __shared__ int2 lists_dyn[];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int W = blockDim.x >> 6;
  const int s = blockIdx.x;
  const int k = a.k, P = a.P;
  const int r0 = a.off[s], r1 = a.off[s + 1];

  if (tid < K2_LS) lists_dyn[tid] = make_int2(kNegInfBits, INT_MAX);
  // running best k of the sentence lives in slots [0, k); empty slots hold
  // distinct keys below every real candidate
  if (tid < k) {
    key[tid] = cand_key(-INFINITY, INT_MAX - tid);
    c_t[tid] = -1;
    c_p[tid] = -1;
  }
  const int wbase = K2_LS + wave * P * K2_LS;  // this wave's lists in lists_dyn
  int lidx[NQ];  // each lane's lists, or the empty list where it has none
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const int p = lane + 64 * q;
    lidx[q] = p < P ? wbase + p * K2_LS : 0;
  }

  for (int cr0 = r0; cr0 < r1; cr0 += W) {
    const int nrows = min(W, r1 - cr0);
    const int ri = wave;
    const bool active = ri < nrows;
    const int r = cr0 + ri;
    float2 st[NQ];
    float prev_r = 0.f;
    if (active) {
      // the row's split statistics and previous score first, so that their
      // loads are in flight with the lists' (one memory round trip for a
      // row whose lists take one batch)
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        const int p = lane + 64 * q;
        st[q] = p < P ? a.stats[(size_t)p * a.N + r] : make_float2(kStatInit, 0.f);
      }
      prev_r = a.prev[r];
      // lane = kp * g + j (kp: k rounded up to a power of two) stages entry j
      // of lists p0 + g, p0 + gpl + g, ... (gpl = 64 / kp lists per load;
      // slots k .. kp - 1 get empty entries): LB loads in flight per lane
      // before the first LDS write (as many as the registers allow: 32 in the
      // 512-thread form, whose row of up to 256 splits then takes one batch
      // up to k = 8; 16, or 8 for the longest split counts, in the 1024-thread
      // form).  Slots past kp are never read before a list has given up all
      // k entries, so they stay unwritten.
      constexpr int LB = MAXT <= 512 ? 32 : (NQ <= 2 ? 16 : 8);
      const int lgk = k <= 1 ? 0 : (k <= 2 ? 1 : (k <= 4 ? 2 : (k <= 8 ? 3 : 4)));
      const int j = lane & ((1 << lgk) - 1), g = lane >> lgk, gpl = 64 >> lgk;
      for (int p0 = 0; p0 < P; p0 += LB * gpl) {
        int2 v[LB];
#pragma unroll
        for (int u = 0; u < LB; ++u) {
          const int p = p0 + u * gpl + g;
          v[u] = make_int2(kNegInfBits, INT_MAX);
          if (p < P && j < k) v[u] = a.lists[((size_t)p * a.N + r) * k + j];
        }
#pragma unroll
        for (int u = 0; u < LB; ++u) {
          const int p = p0 + u * gpl + g;
          if (p < P) lists_dyn[wbase + p * K2_LS + j] = v[u];
        }
      }
    }
    __syncthreads();  // the staged lists are visible; the running best is settled
    uint64_t my_key = cand_key(-INFINITY, INT_MAX - (k + ri * k + lane));
    int my_t = -1;
    if (active) {
      float M = kStatInit;
#pragma unroll
      for (int q = 0; q < NQ; ++q) M = fmaxf(M, st[q].x);
      M = wave_max(M);
      float S = 0.f;
#pragma unroll
      for (int q = 0; q < NQ; ++q) S += st[q].y * __expf(st[q].x - M);
      S = wave_sum(S);
      const float lse = M + __logf(S);
      if (a.row_lse != nullptr && lane == 0) a.row_lse[r] = lse;
      const float base = prev_r - lse;
      const float kth = key_score(key[k - 1]);  // running k-th best (-inf before the first chunk)

      // per list of this lane: the key of its head (entry ptr) and the entry after it
      uint64_t hk[NQ];
      int2 nx[NQ];
      int ptr[NQ];
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        const int2 h = lists_dyn[lidx[q]];
        nx[q] = lists_dyn[lidx[q] + 1];
        hk[q] = key_of(__int_as_float(h.x), h.y);
        ptr[q] = 0;
      }
      for (int jr = 0; jr < k; ++jr) {
        // the wave-wide best head (branch-free: DPP and scalar maxima on keys)
        uint64_t best = hk[0];
#pragma unroll
        for (int q = 1; q < NQ; ++q) best = hk[q] > best ? hk[q] : best;
        const uint64_t win = wave_max64(best);
        const float wv = key_score(win);
        const int wi = key_index(win);
        // the row's later entries are worse still: once this one scores below
        // the sentence's k-th best of the rows ranked so far, none can enter
        if (wv + base < kth) break;
        if (lane == jr && wv > -INFINITY) {
          my_key = cand_key(wv + base, (r - r0) * a.V + wi);
          my_t = wi;
        }
        // the list whose head won advances (words are unique; empty heads
        // are all alike and advance together); every lane then reloads the
        // entry after its heads, so the read is waited for only at the next
        // advance.  A list advances at most once a round, k rounds in all,
        // and its head is compared only while rounds remain, so the clamped
        // read past the last slot is never used.
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
          const bool adv = hk[q] == win;
          hk[q] = adv ? key_of(__int_as_float(nx[q].x), nx[q].y) : hk[q];
          ptr[q] += adv ? 1 : 0;
          nx[q] = lists_dyn[lidx[q] + min(ptr[q] + 1, K2_LS - 1)];
        }
      }
    }
    const int C = k + nrows * k;
    if (active && lane < k) {
      const int slot = k + ri * k + lane;
      key[slot] = my_key;
      c_t[slot] = my_t;
      c_p[slot] = r;
    }
    if (tid == 0 && (C & 1)) key[C] = 0;  // pairs: a pad below every key
    __syncthreads();
    // rank every candidate (running best + this chunk) and keep the first k
    if (tid < C) {
      const uint64_t me = key[tid];
      const ulonglong2* kp = reinterpret_cast<const ulonglong2*>(key);
      int rank = 0;
      const int C2 = (C + 1) >> 1;
#pragma unroll 4
      for (int o = 0; o < C2; ++o) {
        const ulonglong2 q = kp[o];
        rank += (q.x > me ? 1 : 0) + (q.y > me ? 1 : 0);
      }
      if (rank < k) {
        n_key[rank] = me;
        n_t[rank] = c_t[tid];
        n_p[rank] = c_p[tid];
      }
    }
    __syncthreads();
    if (tid < k) {
      key[tid] = n_key[tid];
      c_t[tid] = n_t[tid];
      c_p[tid] = n_p[tid];
    }
    __syncthreads();
  }
  if (tid < k) {
    a.tok[s * k + tid] = c_t[tid];
    a.par[s * k + tid] = c_p[tid];
    a.score[s * k + tid] = key_score(key[tid]);
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
// splits lane, lane + 64, ..., then the wave-wide largest key.  Empty list slots
// hold scores below every real one, and the split holding the row's maximum
// always lists it.
__global__ __launch_bounds__(256) void k2_argmax(const int2* __restrict__ lists, int P, int N,
                                                 int32_t* __restrict__ tok, float* __restrict__ val) {
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= N) return;  // whole waves leave together
  uint64_t best = kEmptyKey;
  for (int p = lane; p < P; p += 64) {
    const int2 e = lists[(size_t)p * N + r];
    const uint64_t key = key_of(__int_as_float(e.x), e.y);
    best = key > best ? key : best;
  }
  best = wave_max64(best);
  if (lane == 0) {
    tok[r] = key_index(best);
    val[r] = key_score(best);
  }
}

hipError_t launch_k2_argmax(const int2* lists, int P, int N, int32_t* tok, float* val, hipStream_t st) {
  if (N <= 0) return hipSuccess;
  k2_argmax<<<dim3((N + 3) / 4), dim3(256), 0, st>>>(lists, P, N, tok, val);
  return hipGetLastError();
}

template <int NQ, int MAXT>
static hipError_t launch_k2_w(const K2Args& a, int W, size_t lds, hipStream_t st) {
  static bool attr_set = false;  // the kernel's LDS ceiling (at most 144 KB + one list), raised once per process
  if (lds > 48 * 1024 && !attr_set) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k2_merge<NQ, MAXT>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize,
                                             (int)(K2_LS * sizeof(int2) + 144 * 1024));
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  k2_merge<NQ, MAXT><<<dim3(a.S), dim3(64 * W), lds, st>>>(a);
  return hipGetLastError();
}

template <int NQ>
static hipError_t launch_k2_nq(const K2Args& a, hipStream_t st) {
  // one wave per row of a sentence of average length (longer sentences take
  // their rows in chunks), as many as the staged lists fit in 144 KB of LDS
  // (the kernel's static LDS is under 4 KB): at most 16 up to P = 72, 4 at P = 256
  const size_t per_wave = (size_t)a.P * K2_LS * sizeof(int2);
  const int rows_per = (a.N + a.S - 1) / a.S;
  const int W = (int)std::min<size_t>(std::min(K2_MAXW, std::max(1, rows_per)), (144 * 1024) / per_wave);
  const size_t lds = (size_t)K2_LS * sizeof(int2) + (size_t)W * per_wave;
  // past 128 splits a row's lists take more than 16 KB, so at most 8 waves fit:
  // only the 512-thread form is built for 3 and 4 lists per lane
  if constexpr (NQ >= 3) {
    return launch_k2_w<NQ, 512>(a, W, lds, st);
  } else {
    // The 512-thread form stages a row's lists in batches of 32 loads per
    // lane against 16, but takes about 210 VGPRs against 125: a CU then holds
    // one workgroup of five waves instead of three.  It is used only where it
    // saves a staging batch (a row's lists past 16 * 64 / kp splits, kp = k
    // rounded up to a power of two) and the sentences need at most one
    // workgroup per CU; with more (512 sentences at 25 splits, say) the
    // 1024-thread form's occupancy halves the merge's time.
    const int kp = a.k <= 1 ? 1 : (a.k <= 2 ? 2 : (a.k <= 4 ? 4 : (a.k <= 8 ? 8 : 16)));
    const int per_batch = 16 * (64 / kp);  // lists of a row per batch of the 1024-thread form
    const bool saves_batch = (a.P + per_batch - 1) / per_batch > (a.P + 2 * per_batch - 1) / (2 * per_batch);
    return W <= 8 && saves_batch && a.S <= 256 ? launch_k2_w<NQ, 512>(a, W, lds, st)
                                               : launch_k2_w<NQ, 1024>(a, W, lds, st);
  }
}

// A vocabulary shard's partial lists hold shard-local words; this moves them
// to the shard's place in the whole vocabulary.  Empty entries (word -1 or
// INT_MAX, score below every real one) keep their word.
__global__ __launch_bounds__(256) void add_word_base(int2* __restrict__ lists, size_t n, int base, int v_shard) {
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (size_t)gridDim.x * 256) {
    const int w = lists[i].y;
    if ((unsigned)w < (unsigned)v_shard) lists[i].y = w + base;
  }
}

hipError_t launch_add_word_base(int2* lists, size_t n, int base, int v_shard, hipStream_t st) {
  if (n == 0 || base == 0) return hipSuccess;
  const int blocks = (int)std::min<size_t>((n + 255) / 256, 2048);
  add_word_base<<<dim3(blocks), dim3(256), 0, st>>>(lists, n, base, v_shard);
  return hipGetLastError();
}

hipError_t launch_k2(const K2Args& a, hipStream_t st) {
  if (a.P < 1 || a.P > 64 * K2_LPL || a.k < 1 || a.k > K2_LS) return hipErrorInvalidValue;
  if (a.S <= 0) return hipSuccess;
  switch ((a.P + 63) / 64) {
    case 1: return launch_k2_nq<1>(a, st);
    case 2: return launch_k2_nq<2>(a, st);
    case 3: return launch_k2_nq<3>(a, st);
    default: return launch_k2_nq<4>(a, st);
  }
}

}  // namespace kb
