// Parts shared by both projection kernels: tile layouts, the sorted k-list,
// and the fused epilogue that turns a tile of logits into softmax statistics
// and k-best candidates without writing the logits anywhere.
#pragma once

#include "kb_common.hpp"

namespace kb {

#define KB_LDS __attribute__((address_space(3)))
typedef short s16x4 __attribute__((ext_vector_type(4)));

// XOR swizzle of the 16-byte chunks of W row r: rows r..r+3 read together by
// one transpose read land on distinct banks.
__device__ __forceinline__ int wswz(int r) { return 4 * (r & 3) + 2 * ((r >> 1) & 1); }

// XOR swizzle of the four 16-byte chunks of an h row: the 16 rows read by a
// 16-lane group at one logical chunk fall on 16 distinct 16-byte bank slots.
__device__ __forceinline__ int hswz(int n) { return (n >> 2) & 3; }

// s_waitcnt vmcnt(n) with expcnt / lgkmcnt left alone (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

template <int WV_, int WH_, int NWV_, int NWH_>
struct Lay {
  static constexpr int WV = WV_;    // 32-wide vocabulary blocks per wave
  static constexpr int WH = WH_;    // 32-wide hypothesis blocks per wave
  static constexpr int NWV = NWV_;  // waves along the vocabulary
  static constexpr int NWH = NWH_;  // waves along the hypotheses
  static_assert(NWV * NWH == 4, "four waves per workgroup");
  static constexpr int BV = 32 * WV * NWV;
  static constexpr int BH = 32 * WH * NWH;
  static constexpr int HOLD = 2 * NWV;  // lanes holding one row's scores of a tile
  // Threshold seed of a split's first tile: maxima of 4-score groups when
  // that gives at most 64 per row, else of 16-score groups.
  static constexpr int SEED_G = (HOLD * WV * 4 <= 64) ? 4 : 16;
  static constexpr int SEEDS = HOLD * WV * (16 / SEED_G);
  static constexpr int CAPL = 8;        // candidate slots per lane and row per round
  static constexpr int RED = (SEEDS > 2 * HOLD) ? SEEDS : 2 * HOLD;
};

// Layouts: (WV, WH, NWV, NWH)
using LayL256 = Lay<4, 2, 1, 4>;  // 128 words x 256 rows per tile
using LayL128 = Lay<4, 2, 2, 2>;  // 256 words x 128 rows
using LayL32 = Lay<4, 1, 4, 1>;   // 512 words x 32 rows (few live rows)
using LayL32M = Lay<2, 1, 4, 1>;  // 256 words x 32 rows (few rows, more vocabulary tiles)
using LayL32S = Lay<1, 1, 4, 1>;  // 128 words x 32 rows (few rows, small vocabulary)
using LayL64 = Lay<2, 1, 2, 2>;   // 128 words x 64 rows (DMA pipeline only, two workgroups per CU)

template <class L>
struct alignas(16) SmemEpi {
  float bias[2][L::BV];     // bias of the current / next vocabulary tile
  uint32_t tgk[2][L::BH];   // shared-threshold keys read at the tile's first stage
  float thr[L::BH];   // row's local threshold: k-th best score so far, or the seed
  int lcnt[256][L::WH];
  int flag[2];        // "some lane overflowed" of the current and the next round
  union {
    int2 buf[256][L::WH][L::CAPL];  // candidates of each lane, per row
    float red[L::BH][L::RED];       // seeds, then the per-holder statistics
  } u;
};

// Order-preserving map of floats to unsigned ints for the shared per-row
// threshold (atomicMax).  0 means "no threshold yet".
__device__ __forceinline__ uint32_t f2key(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float key2f(uint32_t k) {
  if (k == 0u) return kNoThr;
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

// ------------------------------------------------------------ sorted k-list
// Descending (score, word) list in KC register slots.  The first KC - k slots
// hold +inf sentinels that nothing displaces, so the k real entries occupy the
// last k slots and the k-th best is always slot KC - 1 (no runtime register
// indexing).  An insertion bubbles the candidate down and drops the last entry.
template <int KC>
__device__ __forceinline__ void list_init(float (&lv)[KC], int (&li)[KC], int k) {
#pragma unroll
  for (int j = 0; j < KC; ++j) {
    const bool sentinel = j < KC - k;
    lv[j] = sentinel ? INFINITY : -INFINITY;
    li[j] = sentinel ? INT_MIN : INT_MAX;
  }
}

template <int KC>
__device__ __forceinline__ void list_insert(float (&lv)[KC], int (&li)[KC], float cv, int ci) {
#pragma unroll
  for (int j = 0; j < KC; ++j) {
    const bool bt = better(cv, ci, lv[j], li[j]);
    const float tv = lv[j];
    const int tx = li[j];
    lv[j] = bt ? cv : tv;
    li[j] = bt ? ci : tx;
    cv = bt ? tv : cv;
    ci = bt ? tx : ci;
  }
}

__device__ __forceinline__ float quad_max(const f32x16& x, int q) {
  return fmaxf(fmaxf(x[4 * q], x[4 * q + 1]), fmaxf(x[4 * q + 2], x[4 * q + 3]));
}

// ------------------------------------------------------------ the epilogue
// Per lane: running (max, sum) of its scores of each of its WH rows.
// Per owner thread (tid < BH): the row's sorted k best of this split.
template <class L, int KC>
struct Epilogue {
  static constexpr int WV = L::WV, WH = L::WH, NWV = L::NWV;
  static constexpr int DONE = WV * 16;
  float st_m[WH], st_s[WH];
  float lval[KC];
  int lidx[KC];
  float published;  // owner: last value pushed to the shared threshold

  __device__ __forceinline__ void init(SmemEpi<L>& ep, int k) {
    const int tid = threadIdx.x;
    if (tid < L::BH) ep.thr[tid] = kNoThr;
    if (tid < 2) ep.flag[tid] = 0;
#pragma unroll
    for (int hb = 0; hb < WH; ++hb) {
      st_m[hb] = kStatInit;
      st_s[hb] = 0.f;
    }
    list_init<KC>(lval, lidx, k);
    published = kNoThr;
  }

  // Shared threshold of this lane's rows (valid lower bounds of each row's
  // k-th best: k scores of the row are >= it).  Issued early, used in tile().
  // (Raw keys: decoding is deferred to the epilogue so that nothing waits on
  // these loads, which would drain the DMA ring issued before them.)
  __device__ __forceinline__ void load_shared_thr(const K1Args& a, int h0, uint32_t (&tg)[WH]) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wh = wave / NWV, col = lane & 31;
#pragma unroll
    for (int hb = 0; hb < WH; ++hb) {
      const int row = min(h0 + (wh * WH + hb) * 32 + col, a.N - 1);
      tg[hb] = a.share ? __hip_atomic_load(&a.gthr[row], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0u;
    }
  }

  __device__ __forceinline__ void owner_publish(const K1Args& a, int row, float v) {
    if (a.share && row < a.N && v > published) {
      atomicMax(&a.gthr[row], f2key(v));
      published = v;
    }
  }

  // One BV x BH tile of logits in acc (MFMA 32x32 layout: lane holds row
  // (hypothesis) col of each 32-block and 16 vocabulary entries).
  __device__ __forceinline__ void tile(f32x16 (&acc)[WV][WH], SmemEpi<L>& ep, const K1Args& a, int h0, int v0,
                                       bool first, const uint32_t (&tg)[WH], const float* bias) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wv = wave % NWV, wh = wave / NWV;
    const int half = lane >> 5, col = lane & 31;
    const int holder = wv * 2 + half;
    const int k = a.k;

    // ---- bias (Algorithm 3 AddBias, fused) and masking of words >= V
    const bool ragged = (v0 + L::BV > a.V);
#pragma unroll
    for (int vb = 0; vb < WV; ++vb) {
      const int vl = (wv * WV + vb) * 32 + 4 * half;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float4 bb = *reinterpret_cast<const float4*>(&bias[vl + 8 * i]);
#pragma unroll
        for (int hb = 0; hb < WH; ++hb) {
          acc[vb][hb][4 * i + 0] += bb.x;
          acc[vb][hb][4 * i + 1] += bb.y;
          acc[vb][hb][4 * i + 2] += bb.z;
          acc[vb][hb][4 * i + 3] += bb.w;
        }
      }
      if (ragged) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int v = v0 + vl + 8 * (r >> 2) + (r & 3);
#pragma unroll
          for (int hb = 0; hb < WH; ++hb)
            if (v >= a.V) acc[vb][hb][r] = -INFINITY;
        }
      }
    }
    // ---- running softmax statistics: one rescale per tile (Algorithm 4's
    // sum <- e^(max_old - max_new) * sum, then the new terms)
#pragma unroll
    for (int hb = 0; hb < WH; ++hb) {
      float m0 = acc[0][hb][0], m1 = acc[0][hb][1];
#pragma unroll
      for (int vb = 0; vb < WV; ++vb)
#pragma unroll
        for (int r = (vb == 0 ? 2 : 0); r < 16; r += 2) {
          m0 = fmaxf(m0, acc[vb][hb][r]);
          m1 = fmaxf(m1, acc[vb][hb][r + 1]);
        }
      const float mnew = fmaxf(st_m[hb], fmaxf(m0, m1));
      const float ml2 = mnew * kL2E;
      float sum = st_s[hb] * exp2_fast((st_m[hb] - mnew) * kL2E);
#pragma unroll
      for (int vb = 0; vb < WV; ++vb)
#pragma unroll
        for (int r = 0; r < 16; ++r) sum += exp2_fast(fmaf(acc[vb][hb][r], kL2E, -ml2));
      st_s[hb] = sum;
      st_m[hb] = mnew;
    }

    // ---- first tile of the split: seed each row's threshold with the k-th
    // largest group maximum (k distinct scores are >= it)
    if (first) {
#pragma unroll
      for (int hb = 0; hb < WH; ++hb) {
        const int hl = (wh * WH + hb) * 32 + col;
#pragma unroll
        for (int vb = 0; vb < WV; ++vb) {
          float qx[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) qx[q] = quad_max(acc[vb][hb], q);
          if constexpr (L::SEED_G == 16) {
            ep.u.red[hl][holder * WV + vb] = fmaxf(fmaxf(qx[0], qx[1]), fmaxf(qx[2], qx[3]));
          } else {
#pragma unroll
            for (int q = 0; q < 4; ++q) ep.u.red[hl][(holder * WV + vb) * 4 + q] = qx[q];
          }
        }
      }
      lds_barrier();
      if (tid < L::BH) {
        float sv[KC];  // right-aligned like the lists: +inf sentinels, then k values
#pragma unroll
        for (int j = 0; j < KC; ++j) sv[j] = (j < KC - k) ? INFINITY : -INFINITY;
        for (int g = 0; g < L::SEEDS; ++g) {
          float x = ep.u.red[tid][g];
#pragma unroll
          for (int j = 0; j < KC; ++j) {
            const float hi = fmaxf(sv[j], x);
            x = fminf(sv[j], x);
            sv[j] = hi;
          }
        }
        const float kth = sv[KC - 1];
        if (kth > ep.thr[tid]) {
          ep.thr[tid] = kth;
          owner_publish(a, h0 + tid, kth);
        }
      }
      lds_barrier();
    }

    // ---- candidate rounds.  A lane appends, in position order, every score
    // >= max(row's local threshold, shared threshold) to its own LDS slots
    // (ties are kept; the owner settles them by word index).  If its slots
    // fill up, the rest waits (by position) for another round.
    int resume[WH];
#pragma unroll
    for (int hb = 0; hb < WH; ++hb) resume[hb] = 0;
    for (int round = 0;; ++round) {
      int ovf = 0;
#pragma unroll
      for (int hb = 0; hb < WH; ++hb) {
        const int hl = (wh * WH + hb) * 32 + col;
        int c = 0;
        if (resume[hb] < DONE) {
          const float t = fmaxf(ep.thr[hl], key2f(tg[hb]));
          const int rs = resume[hb];
          int newres = DONE;
#pragma unroll
          for (int vb = 0; vb < WV; ++vb) {
            const int vbase = v0 + (wv * WV + vb) * 32 + 4 * half;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              if (quad_max(acc[vb][hb], q) >= t && vb * 16 + 4 * q + 3 >= rs) {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                  const int pos = vb * 16 + 4 * q + j;
                  const float x = acc[vb][hb][4 * q + j];
                  if (x >= t && pos >= rs) {
                    if (c < L::CAPL)
                      ep.u.buf[tid][hb][c] = make_int2(__float_as_int(x), vbase + 8 * q + j);
                    else if (newres == DONE)
                      newres = pos;
                    ++c;
                  }
                }
              }
            }
          }
          resume[hb] = newres;
          ovf |= (newres != DONE);
        }
        ep.lcnt[tid][hb] = min(c, L::CAPL);
      }
      if (ovf) ep.flag[round & 1] = 1;
      lds_barrier();
      if (tid == 0) ep.flag[(round + 1) & 1] = 0;  // read only after the next barrier
      if (tid < L::BH) {
        const int hl = tid;
        const int owh = hl / (32 * WH), ohb = (hl / 32) % WH, ocol = hl % 32;
#pragma unroll
        for (int hd = 0; hd < L::HOLD; ++hd) {
          const int htid = (owh * NWV + (hd >> 1)) * 64 + (hd & 1) * 32 + ocol;
          const int c = ep.lcnt[htid][ohb];
          for (int i = 0; i < c; ++i) {
            const int2 e = ep.u.buf[htid][ohb][i];
            const float cv = __int_as_float(e.x);
            if (better(cv, e.y, lval[KC - 1], lidx[KC - 1])) list_insert<KC>(lval, lidx, cv, e.y);
          }
        }
        if (lval[KC - 1] > ep.thr[hl]) {
          ep.thr[hl] = lval[KC - 1];
          owner_publish(a, h0 + hl, lval[KC - 1]);
        }
      }
      lds_barrier();
      if (ep.flag[round & 1] == 0) break;
    }
  }

  // Merge the holders' statistics and write this split's partial of each row.
  __device__ __forceinline__ void finish(SmemEpi<L>& ep, const K1Args& a, int h0, int split) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wv = wave % NWV, wh = wave / NWV;
    const int half = lane >> 5, col = lane & 31;
    const int holder = wv * 2 + half;
    const int k = a.k;
    __syncthreads();
#pragma unroll
    for (int hb = 0; hb < WH; ++hb) {
      const int hl = (wh * WH + hb) * 32 + col;
      ep.u.red[hl][2 * holder + 0] = st_m[hb];
      ep.u.red[hl][2 * holder + 1] = st_s[hb];
    }
    __syncthreads();
    if (tid < L::BH && h0 + tid < a.N) {
      float M = kStatInit;
#pragma unroll
      for (int i = 0; i < L::HOLD; ++i) M = fmaxf(M, ep.u.red[tid][2 * i]);
      float S = 0.f;
#pragma unroll
      for (int i = 0; i < L::HOLD; ++i)
        S += ep.u.red[tid][2 * i + 1] * exp2_fast((ep.u.red[tid][2 * i] - M) * kL2E);
      const size_t row = (size_t)split * a.N + h0 + tid;
      a.stats[row] = make_float2(M, S);
#pragma unroll
      for (int j = 0; j < KC; ++j)
        if (j >= KC - k) a.lists[row * k + (j - (KC - k))] = make_int2(__float_as_int(lval[j]), lidx[j]);
    }
  }
};

}  // namespace kb
