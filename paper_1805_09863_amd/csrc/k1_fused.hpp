// K1: fused output-layer projection for gfx950.
//
// One workgroup owns BH hypothesis rows and a contiguous range of BV-wide
// vocabulary tiles (a "split", the shard of Algorithm 6).  For each tile it
//   1. computes the BV x BH block of x = W^T h^T on the matrix cores
//      (MFMA 32x32, bf16 x bf16 or f32 x f32 products, f32 accumulate;
//      Section 2.2 step 1, half precision per Section 2.3);
//   2. adds the bias in registers (step 2, Algorithm 3 AddBias);
//   3. updates per-row running softmax statistics -- a running max and a sum
//      of exp(x - max) rescaled by exp(max_old - max_new) whenever the max
//      grows (Algorithm 4 and the identity derived after it), one rescale per
//      tile instead of per element;
//   4. keeps the k best (score, word) pairs of each row (Algorithm 4's best
//      search extended to k): scores are tested against the row's current
//      k-th best; the few that pass go through a per-row LDS queue to the
//      thread that owns the row's sorted list.
// The N x V scores never leave registers.  Each split writes one partial per
// row: (max, sum) and its k best pairs; K2 merges the splits.
#pragma once

#include "kb_common.hpp"

namespace kb {

template <int WV_, int WH_, int NWV_, int NWH_, int CAP_>
struct Lay {
  static constexpr int WV = WV_;    // 32-wide vocabulary blocks per wave
  static constexpr int WH = WH_;    // 32-wide hypothesis blocks per wave
  static constexpr int NWV = NWV_;  // waves along the vocabulary
  static constexpr int NWH = NWH_;  // waves along the hypotheses
  static_assert(NWV * NWH == 4, "four waves per workgroup");
  static constexpr int BV = 32 * WV * NWV;
  static constexpr int BH = 32 * WH * NWH;
  static constexpr int HOLD = 2 * NWV;      // lanes holding one row's scores of a tile
  // Threshold seed of a split's first tile: maxima of 4-score groups when
  // that gives at most 64 per row, else of 16-score groups.
  static constexpr int SEED_G = (HOLD * WV * 4 <= 64) ? 4 : 16;
  static constexpr int SEEDS = HOLD * WV * (16 / SEED_G);
  static constexpr int CAP = CAP_;          // candidate queue slots per row
  static constexpr int RED = (SEEDS > 2 * HOLD) ? SEEDS : 2 * HOLD;
};

template <bool BF16>
struct Ty;
template <>
struct Ty<true> {
  using E = uint16_t;
  static constexpr int BK = 64;   // K per LDS stage
  static constexpr int KM = 16;   // K per MFMA
  static constexpr int VEC = 8;   // elements per 16-byte vector
};
template <>
struct Ty<false> {
  using E = float;
  static constexpr int BK = 32;
  static constexpr int KM = 2;
  static constexpr int VEC = 4;
};

// LDS.  bf16: both operands K-contiguous ([row][k]) so every MFMA fragment is
// one 16-byte read; W arrives V-contiguous and is transposed in registers.
// f32: one element per lane per operand, stored [k][row] without transposing.
template <bool BF16, class L>
struct Smem;

template <class L>
struct SmemEpi {
  float bias[L::BV];
  float thr[L::BH];
  int thri[L::BH];
  int cnt[L::BH];
  int2 q[L::BH][L::CAP];
  float red[L::BH][L::RED];
};

template <class L>
struct Smem<true, L> {
  static constexpr int P = Ty<true>::BK + 8;
  uint16_t Ws[L::BV][P];
  uint16_t Hs[L::BH][P];
  SmemEpi<L> e;
};

template <class L>
struct Smem<false, L> {
  uint32_t Ws[Ty<false>::BK][L::BV + 4];
  uint32_t Hs[Ty<false>::BK][L::BH + 4];
  SmemEpi<L> e;
};

// ------------------------------------------------------------ global -> regs
template <bool BF16, class L>
struct Stage {
  using T = Ty<BF16>;
  static constexpr int BK = T::BK;
  // bf16: h chunks of 8 k; W blocks of 8k x 8v.  f32: h chunks of 4 k; W chunks of 4 v.
  static constexpr int H_CHUNKS = L::BH * BK / T::VEC;
  static constexpr int W_UNITS = BF16 ? (BK / 8) * (L::BV / 8) : BK * L::BV / 4;
  static constexpr int H_PER = (H_CHUNKS + 255) / 256;
  static constexpr int W_PER = (W_UNITS + 255) / 256;
  static constexpr int W_ROWS = BF16 ? 8 : 1;  // 16-byte rows per W unit
  uint4 hv[H_PER];
  uint4 wv[W_PER][W_ROWS];
};

template <bool BF16>
__device__ __forceinline__ uint4 load_vec_guarded(const void* base, size_t row_elems, int row, int col,
                                                  int nrows, int ncols, bool vec_ok) {
  using E = typename Ty<BF16>::E;
  constexpr int VEC = Ty<BF16>::VEC;
  const E* p = reinterpret_cast<const E*>(base);
  uint4 r = make_uint4(0, 0, 0, 0);
  if (row >= nrows || col >= ncols) return r;
  const size_t off = (size_t)row * row_elems + (size_t)col;
  if (vec_ok) return *reinterpret_cast<const uint4*>(p + off);
  E tmp[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) tmp[e] = (col + e < ncols) ? p[off + e] : E(0);
  __builtin_memcpy(&r, tmp, 16);
  return r;
}

template <bool BF16, class L>
__device__ __forceinline__ void stage_load(Stage<BF16, L>& s, const K1Args& a, int h0, int v0, int k0,
                                           int tid) {
  using S = Stage<BF16, L>;
  constexpr int BK = S::BK;
  const bool vec = a.vec_ok != 0;
#pragma unroll
  for (int i = 0; i < S::H_PER; ++i) {
    const int c = tid + 256 * i;
    if (S::H_CHUNKS % 256 == 0 || c < S::H_CHUNKS) {
      int n, kc;
      if (BF16) {
        n = c / (BK / 8);
        kc = (c % (BK / 8)) * 8;
      } else {
        kc = (c / L::BH) * 4;
        n = c % L::BH;
      }
      s.hv[i] = load_vec_guarded<BF16>(a.h, (size_t)a.H, h0 + n, k0 + kc, a.N, a.H, vec);
    }
  }
#pragma unroll
  for (int i = 0; i < S::W_PER; ++i) {
    const int u = tid + 256 * i;
    if (S::W_UNITS % 256 == 0 || u < S::W_UNITS) {
      if (BF16) {
        const int kb = u / (L::BV / 8), vc = u % (L::BV / 8);
#pragma unroll
        for (int r = 0; r < 8; ++r)
          s.wv[i][r] = load_vec_guarded<true>(a.W, (size_t)a.V, k0 + kb * 8 + r, v0 + vc * 8, a.H, a.V, vec);
      } else {
        const int kr = u / (L::BV / 4), vc = u % (L::BV / 4);
        s.wv[i][0] = load_vec_guarded<false>(a.W, (size_t)a.V, k0 + kr, v0 + vc * 4, a.H, a.V, vec);
      }
    }
  }
}

// 16-bit halves of a 32-bit word
__device__ __forceinline__ uint32_t lo16(uint32_t w) { return w & 0xFFFFu; }
__device__ __forceinline__ uint32_t hi16(uint32_t w) { return w >> 16; }
__device__ __forceinline__ uint32_t word(const uint4& v, int i) {
  return i == 0 ? v.x : (i == 1 ? v.y : (i == 2 ? v.z : v.w));
}

template <bool BF16, class L>
__device__ __forceinline__ void stage_store(const Stage<BF16, L>& s, Smem<BF16, L>& sm, int tid) {
  using S = Stage<BF16, L>;
  constexpr int BK = S::BK;
#pragma unroll
  for (int i = 0; i < S::H_PER; ++i) {
    const int c = tid + 256 * i;
    if (S::H_CHUNKS % 256 == 0 || c < S::H_CHUNKS) {
      if (BF16) {
        const int n = c / (BK / 8), kc = (c % (BK / 8)) * 8;
        *reinterpret_cast<uint4*>(&sm.Hs[n][kc]) = s.hv[i];
      } else {
        const int kc = (c / L::BH) * 4, n = c % L::BH;
        sm.Hs[kc + 0][n] = s.hv[i].x;
        sm.Hs[kc + 1][n] = s.hv[i].y;
        sm.Hs[kc + 2][n] = s.hv[i].z;
        sm.Hs[kc + 3][n] = s.hv[i].w;
      }
    }
  }
#pragma unroll
  for (int i = 0; i < S::W_PER; ++i) {
    const int u = tid + 256 * i;
    if (S::W_UNITS % 256 == 0 || u < S::W_UNITS) {
      if (BF16) {
        // 8 (k) x 8 (v) block: rows r of s.wv hold v = vc*8 .. vc*8+7 at k = kb*8 + r.
        // Column c of the block becomes one K-contiguous 16-byte LDS row.
        const int kb = u / (L::BV / 8), vc = u % (L::BV / 8);
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          uint32_t o[4];
#pragma unroll
          for (int p = 0; p < 4; ++p) {
            const uint32_t a0 = word(s.wv[i][2 * p], c >> 1);
            const uint32_t a1 = word(s.wv[i][2 * p + 1], c >> 1);
            o[p] = (c & 1) ? (hi16(a0) | (a1 & 0xFFFF0000u)) : (lo16(a0) | (a1 << 16));
          }
          *reinterpret_cast<uint4*>(&sm.Ws[vc * 8 + c][kb * 8]) = make_uint4(o[0], o[1], o[2], o[3]);
        }
      } else {
        const int kr = u / (L::BV / 4), vc = u % (L::BV / 4);
        *reinterpret_cast<uint4*>(&sm.Ws[kr][vc * 4]) = s.wv[i][0];
      }
    }
  }
}

// ------------------------------------------------------------ MFMA stage
template <bool BF16, class L>
__device__ __forceinline__ void stage_mma(f32x16 (&acc)[L::WV][L::WH], const Smem<BF16, L>& sm, int wv,
                                          int wh, int lane) {
  constexpr int BK = Ty<BF16>::BK;
  const int half = lane >> 5, col = lane & 31;
  if constexpr (BF16) {
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      bf16x8 af[L::WV], bf[L::WH];
#pragma unroll
      for (int vb = 0; vb < L::WV; ++vb)
        af[vb] = *reinterpret_cast<const bf16x8*>(&sm.Ws[(wv * L::WV + vb) * 32 + col][kk * 16 + half * 8]);
#pragma unroll
      for (int hb = 0; hb < L::WH; ++hb)
        bf[hb] = *reinterpret_cast<const bf16x8*>(&sm.Hs[(wh * L::WH + hb) * 32 + col][kk * 16 + half * 8]);
#pragma unroll
      for (int vb = 0; vb < L::WV; ++vb)
#pragma unroll
        for (int hb = 0; hb < L::WH; ++hb)
          acc[vb][hb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[vb], bf[hb], acc[vb][hb], 0, 0, 0);
    }
  } else {
#pragma unroll
    for (int kk = 0; kk < BK / 2; ++kk) {
      float af[L::WV], bf[L::WH];
#pragma unroll
      for (int vb = 0; vb < L::WV; ++vb)
        af[vb] = __uint_as_float(sm.Ws[kk * 2 + half][(wv * L::WV + vb) * 32 + col]);
#pragma unroll
      for (int hb = 0; hb < L::WH; ++hb)
        bf[hb] = __uint_as_float(sm.Hs[kk * 2 + half][(wh * L::WH + hb) * 32 + col]);
#pragma unroll
      for (int vb = 0; vb < L::WV; ++vb)
#pragma unroll
        for (int hb = 0; hb < L::WH; ++hb)
          acc[vb][hb] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[vb], bf[hb], acc[vb][hb], 0, 0, 0);
    }
  }
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

// ------------------------------------------------------------ the kernel
template <bool BF16, class L, int KC>
__global__ __launch_bounds__(256) void k1_fused(K1Args a) {
  constexpr int BK = Ty<BF16>::BK;
  constexpr int BV = L::BV, BH = L::BH, WV = L::WV, WH = L::WH;
  constexpr int DONE = WV * 16;
  __shared__ Smem<BF16, L> sm;
  SmemEpi<L>& ep = sm.e;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wv = wave % L::NWV, wh = wave / L::NWV;
  const int half = lane >> 5, col = lane & 31;
  const int holder = wv * 2 + half;
  const int split = blockIdx.x;
  const int h0 = blockIdx.y * BH;
  const int vt0 = split * a.tps;
  const int vt1 = min(vt0 + a.tps, a.n_vtiles);
  const int nk = (a.H + BK - 1) / BK;
  const int k = a.k;

  if (tid < BH) {
    ep.thr[tid] = kNoThr;
    ep.thri[tid] = INT_MAX;
    ep.cnt[tid] = 0;
  }
  // owner state: thread tid < BH owns row h0 + tid of this workgroup
  float lval[KC];
  int lidx[KC];
  list_init<KC>(lval, lidx, k);
  // holder state: running (max, sum) of this lane's scores for each of its WH rows
  float st_m[WH], st_s[WH];
#pragma unroll
  for (int hb = 0; hb < WH; ++hb) {
    st_m[hb] = kStatInit;
    st_s[hb] = 0.f;
  }

  Stage<BF16, L> pf;
  stage_load<BF16, L>(pf, a, h0, vt0 * BV, 0, tid);

  for (int vt = vt0; vt < vt1; ++vt) {
    const int v0 = vt * BV;
    f32x16 acc[WV][WH];
#pragma unroll
    for (int vb = 0; vb < WV; ++vb)
#pragma unroll
      for (int hb = 0; hb < WH; ++hb)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[vb][hb][r] = 0.f;

    for (int kt = 0; kt < nk; ++kt) {
      __syncthreads();
      stage_store<BF16, L>(pf, sm, tid);
      if (kt == 0)
        for (int i = tid; i < BV; i += 256) ep.bias[i] = (v0 + i < a.V) ? a.b[v0 + i] : 0.f;
      __syncthreads();
      if (kt + 1 < nk) stage_load<BF16, L>(pf, a, h0, v0, (kt + 1) * BK, tid);
      stage_mma<BF16, L>(acc, sm, wv, wh, lane);
    }

    // ---------------- epilogue: bias, group maxima, softmax statistics
    const bool ragged = (v0 + BV > a.V);
    float gm[WV][WH];
#pragma unroll
    for (int vb = 0; vb < WV; ++vb) {
      const int vl = (wv * WV + vb) * 32 + 4 * half;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float4 bb = *reinterpret_cast<const float4*>(&ep.bias[vl + 8 * i]);
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
#pragma unroll
      for (int hb = 0; hb < WH; ++hb) {
        float m0 = fmaxf(acc[vb][hb][0], acc[vb][hb][1]);
        float m1 = fmaxf(acc[vb][hb][2], acc[vb][hb][3]);
#pragma unroll
        for (int r = 4; r < 16; r += 2) {
          m0 = fmaxf(m0, acc[vb][hb][r]);
          m1 = fmaxf(m1, acc[vb][hb][r + 1]);
        }
        gm[vb][hb] = fmaxf(m0, m1);
      }
    }
#pragma unroll
    for (int hb = 0; hb < WH; ++hb) {
      float tmax = gm[0][hb];
#pragma unroll
      for (int vb = 1; vb < WV; ++vb) tmax = fmaxf(tmax, gm[vb][hb]);
      const float mnew = fmaxf(st_m[hb], tmax);
      const float ml2 = mnew * kL2E;
      float sum = st_s[hb] * exp2_fast((st_m[hb] - mnew) * kL2E);
#pragma unroll
      for (int vb = 0; vb < WV; ++vb)
#pragma unroll
        for (int r = 0; r < 16; ++r) sum += exp2_fast(fmaf(acc[vb][hb][r], kL2E, -ml2));
      st_s[hb] = sum;
      st_m[hb] = mnew;
    }

    // ---------------- first tile of the split: seed each row's threshold with
    // the k-th largest group maximum (k distinct scores are >= it).
    if (vt == vt0) {
#pragma unroll
      for (int hb = 0; hb < WH; ++hb) {
        const int hl = (wh * WH + hb) * 32 + col;
#pragma unroll
        for (int vb = 0; vb < WV; ++vb) {
          if constexpr (L::SEED_G == 16) {
            ep.red[hl][holder * WV + vb] = gm[vb][hb];
          } else {
#pragma unroll
            for (int q = 0; q < 4; ++q)
              ep.red[hl][(holder * WV + vb) * 4 + q] =
                  fmaxf(fmaxf(acc[vb][hb][4 * q], acc[vb][hb][4 * q + 1]),
                        fmaxf(acc[vb][hb][4 * q + 2], acc[vb][hb][4 * q + 3]));
          }
        }
      }
      __syncthreads();
      if (tid < BH) {
        float sv[KC];  // right-aligned like the lists: +inf sentinels, then k values
#pragma unroll
        for (int j = 0; j < KC; ++j) sv[j] = (j < KC - k) ? INFINITY : -INFINITY;
        for (int g = 0; g < L::SEEDS; ++g) {
          float x = ep.red[tid][g];
#pragma unroll
          for (int j = 0; j < KC; ++j) {
            const float hi = fmaxf(sv[j], x);
            x = fminf(sv[j], x);
            sv[j] = hi;
          }
        }
        const float kth = sv[KC - 1];
        if (kth > -INFINITY) {
          ep.thr[tid] = kth;
          ep.thri[tid] = INT_MAX;  // scores equal to the seed still pass
        }
      }
      __syncthreads();
    }

    // ---------------- candidate rounds: scores beating the row's k-th best
    // go to the row's queue; the owner merges them.  A full queue defers the
    // rest of that lane's scores (by position) to another round.
    int resume[WH];
#pragma unroll
    for (int hb = 0; hb < WH; ++hb) resume[hb] = 0;
    while (true) {
      int ovf = 0;
#pragma unroll
      for (int hb = 0; hb < WH; ++hb) {
        const int hl = (wh * WH + hb) * 32 + col;
        if (resume[hb] < DONE) {
          const float t = ep.thr[hl];
          const int ti = ep.thri[hl];
          const int rs = resume[hb];
          int newres = DONE;
#pragma unroll
          for (int vb = 0; vb < WV; ++vb) {
            if (newres == DONE && gm[vb][hb] >= t && vb * 16 + 15 >= rs) {
              const int vbase = v0 + (wv * WV + vb) * 32 + 4 * half;
              int c = 0;
#pragma unroll
              for (int r = 0; r < 16; ++r) {
                const int v = vbase + 8 * (r >> 2) + (r & 3);
                const float x = acc[vb][hb][r];
                c += (vb * 16 + r >= rs && better(x, v, t, ti)) ? 1 : 0;
              }
              if (c) {
                int o = atomicAdd(&ep.cnt[hl], c);
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                  const int v = vbase + 8 * (r >> 2) + (r & 3);
                  const float x = acc[vb][hb][r];
                  if (vb * 16 + r >= rs && better(x, v, t, ti)) {
                    if (o < L::CAP)
                      ep.q[hl][o] = make_int2(__float_as_int(x), v);
                    else if (newres == DONE)
                      newres = vb * 16 + r;
                    ++o;
                  }
                }
              }
            }
          }
          resume[hb] = newres;
          ovf |= (newres != DONE);
        }
      }
      __syncthreads();
      if (tid < BH) {
        const int c = min(ep.cnt[tid], L::CAP);
        for (int i = 0; i < c; ++i) {
          const int2 e = ep.q[tid][i];
          const float cv = __int_as_float(e.x);
          if (better(cv, e.y, lval[KC - 1], lidx[KC - 1])) list_insert<KC>(lval, lidx, cv, e.y);
        }
        ep.cnt[tid] = 0;
        if (lval[KC - 1] > -INFINITY) {
          ep.thr[tid] = lval[KC - 1];
          ep.thri[tid] = lidx[KC - 1];
        }
      }
      if (!__syncthreads_or(ovf)) break;
    }
    if (vt + 1 < vt1) stage_load<BF16, L>(pf, a, h0, v0 + BV, 0, tid);
  }

  // ---------------- write this split's partial for every row it owns
#pragma unroll
  for (int hb = 0; hb < WH; ++hb) {
    const int hl = (wh * WH + hb) * 32 + col;
    ep.red[hl][2 * holder + 0] = st_m[hb];
    ep.red[hl][2 * holder + 1] = st_s[hb];
  }
  __syncthreads();
  if (tid < BH && h0 + tid < a.N) {
    float M = kStatInit;
#pragma unroll
    for (int i = 0; i < L::HOLD; ++i) M = fmaxf(M, ep.red[tid][2 * i]);
    float S = 0.f;
#pragma unroll
    for (int i = 0; i < L::HOLD; ++i) S += ep.red[tid][2 * i + 1] * exp2_fast((ep.red[tid][2 * i] - M) * kL2E);
    const size_t row = (size_t)split * a.N + h0 + tid;
    a.stats[row] = make_float2(M, S);
#pragma unroll
    for (int j = 0; j < KC; ++j)
      if (j >= KC - k) a.lists[row * k + (j - (KC - k))] = make_int2(__float_as_int(lval[j]), lidx[j]);
  }
}

// Layouts: (WV, WH, NWV, NWH, CAP)
using LayL256 = Lay<4, 2, 1, 4, 24>;  // 128 words x 256 rows per tile
using LayL128 = Lay<4, 2, 2, 2, 24>;  // 256 words x 128 rows
using LayL32 = Lay<4, 1, 4, 1, 32>;   // 512 words x 32 rows (few live rows)

template <bool BF16, class L>
hipError_t launch_k1_layout(int kc, dim3 grid, const K1Args& a, hipStream_t st) {
  const dim3 block(256);
  switch (kc) {
    case 4: k1_fused<BF16, L, 4><<<grid, block, 0, st>>>(a); break;
    case 8: k1_fused<BF16, L, 8><<<grid, block, 0, st>>>(a); break;
    case 12: k1_fused<BF16, L, 12><<<grid, block, 0, st>>>(a); break;
    case 16: k1_fused<BF16, L, 16><<<grid, block, 0, st>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace kb
