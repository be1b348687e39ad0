// K1, register-staged variant: fused output-layer projection for gfx950 that
// handles every shape (float32 or bf16, any H and V, any alignment).
//
// One workgroup owns BH hypothesis rows and a contiguous range of BV-wide
// vocabulary tiles (a "split", the shard of Algorithm 6).  For each tile it
//   1. computes the BV x BH block of x = W^T h^T on the matrix cores
//      (MFMA 32x32, bf16 x bf16 or f32 x f32 products, f32 accumulate;
//      Section 2.2 step 1, half precision per Section 2.3); operands go
//      global -> registers -> LDS, bf16 W transposed in registers so both
//      operands are K-contiguous in LDS;
//   2. runs the fused epilogue (k1_common.hpp): bias, softmax statistics and
//      the split's k best words of every row.
// The N x V scores never leave registers.
#pragma once

#include "k1_common.hpp"

namespace kb {

template <bool BF16>
struct Ty;
template <>
struct Ty<true> {
  using E = uint16_t;
  static constexpr int BK = 32;   // K per LDS stage
  static constexpr int VEC = 8;   // elements per 16-byte vector
};
template <>
struct Ty<false> {
  using E = float;
  static constexpr int BK = 32;
  static constexpr int VEC = 4;
};

// LDS.  bf16: both operands K-contiguous ([row][k]) so every MFMA fragment is
// one 16-byte read; W arrives V-contiguous and is transposed in registers.
// f32: one element per lane per operand, stored [k][row] without transposing.
template <bool BF16, class L>
struct SmemReg;

template <class L>
struct SmemReg<true, L> {
  static constexpr int P = Ty<true>::BK + 8;
  uint16_t Ws[L::BV][P];
  uint16_t Hs[L::BH][P];
  SmemEpi<L> e;
};

template <class L>
struct SmemReg<false, L> {
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

__device__ __forceinline__ uint32_t word(const uint4& v, int i) {
  return i == 0 ? v.x : (i == 1 ? v.y : (i == 2 ? v.z : v.w));
}

template <bool BF16, class L>
__device__ __forceinline__ void stage_store(const Stage<BF16, L>& s, SmemReg<BF16, L>& sm, int tid) {
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
            o[p] = (c & 1) ? ((a0 >> 16) | (a1 & 0xFFFF0000u)) : ((a0 & 0xFFFFu) | (a1 << 16));
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
__device__ __forceinline__ void stage_mma(f32x16 (&acc)[L::WV][L::WH], const SmemReg<BF16, L>& sm, int wv,
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

// ------------------------------------------------------------ the kernel
template <bool BF16, class L, int KC>
__global__ __launch_bounds__(256) void k1_fused(K1Args a) {
  constexpr int BK = Ty<BF16>::BK;
  constexpr int BV = L::BV, BH = L::BH, WV = L::WV, WH = L::WH;
  __shared__ __attribute__((aligned(16))) SmemReg<BF16, L> sm;
  SmemEpi<L>& ep = sm.e;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wv = wave % L::NWV, wh = wave / L::NWV;
  int row_tile, split;
  k1_cell(a, blockIdx.x, row_tile, split);
  const int h0 = row_tile * BH;
  const int vt0 = split * a.tps;
  const int vt1 = min(vt0 + a.tps, a.n_vtiles);
  const int nk = (a.H + BK - 1) / BK;

  Epilogue<L, KC> epi;
  epi.init(ep, a.k);

  Stage<BF16, L> pf;
  stage_load<BF16, L>(pf, a, h0, vt0 * BV, 0, tid);

  for (int vt = vt0; vt < vt1; ++vt) {
    const int v0 = vt * BV;
    uint32_t tg[WH];
    epi.load_shared_thr(a, h0, tg);
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
        for (int i = tid; i < BV; i += 256) ep.bias[0][i] = (v0 + i < a.V) ? a.b[v0 + i] : 0.f;
      __syncthreads();
      if (kt + 1 < nk) stage_load<BF16, L>(pf, a, h0, v0, (kt + 1) * BK, tid);
      stage_mma<BF16, L>(acc, sm, wv, wh, lane);
    }
    epi.tile(acc, ep, a, h0, v0, vt == vt0, tg, ep.bias[0]);
    if (vt + 1 < vt1) stage_load<BF16, L>(pf, a, h0, v0 + BV, 0, tid);
  }
  epi.finish(ep, a, h0, split);
}

template <bool BF16, class L>
hipError_t launch_k1_reg(int kc, dim3 grid, const K1Args& a, hipStream_t st) {
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
