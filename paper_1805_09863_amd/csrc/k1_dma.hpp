// K1, DMA variant: the fused output-layer projection for 16-byte aligned
// operands, bf16 h and W with H % 128 == 0 and V % 8 == 0, or float32 with
// H % 64 == 0 and V % 4 == 0.
//
// Same work split and epilogue as the register-staged kernel; the difference
// is how operands reach the matrix cores.  A ring of NS LDS stages (BK = 32
// of the state dimension each) is filled by the gfx950 global->LDS DMA
// (global_load_lds_dwordx4), so loads need no VGPRs and several stages are
// in flight while the MFMAs consume another:
//   * W keeps its V-contiguous layout in LDS; each 16-byte chunk of a row is
//     XOR-swizzled by the row index, and MFMA A-fragments (8 consecutive k
//     of one word) are built with the LDS transpose read ds_read_b64_tr_b16;
//   * h rows are stored row-major, 64 bytes (BK = 32 states) per row, with
//     the four 16-byte chunks XOR-swizzled by row; one DMA instruction reads
//     16 rows x 64 contiguous bytes, and B-fragment reads stay conflict-free.
// Float32 (the fp32 MFMA 32x32x2): a stage holds BK = 16 states, the same
// bytes per row of h (so the same h layout and swizzle) and 16 rows of W
// stored as they arrive (a wave's A-fragment reads, 32 consecutive words of
// one state per half-wave, need no swizzle).  Each lane takes its 16-byte
// chunk of a row of h at once and feeds its 4 states to 4 consecutive
// products: product step s of a stage pairs states 8 * (lane / 32) + s across
// both operands, a fixed permutation of the stage's states, so the sums are
// the same.
// Each stage has its own __shared__ array, which lets the compiler see that
// MFMA-side LDS reads never alias the DMA writes still in flight; the kernel
// waits on the vector-memory counter itself (s_waitcnt vmcnt).
#pragma once

#include <type_traits>

#include "k1_common.hpp"

namespace kb {

template <class L, bool F32>
struct DmaGeom {
  static constexpr int BK = F32 ? 16 : 32;      // K per stage: 64 bytes of an h row
  static constexpr int EPC = F32 ? 4 : 8;       // elements per 16-byte chunk
  static constexpr int NS = 4;                  // stages in the ring
  static constexpr int WCH = L::BV / EPC;       // 16-byte chunks per W row
  static constexpr int W_SLOTS = BK * WCH;      // 16-byte chunks of W per stage
  static constexpr int H_SLOTS = L::BH * 4;    // four 16-byte chunks per h row
  static constexpr int W_PER_WAVE = W_SLOTS / 4;
  static constexpr int H_PER_WAVE = H_SLOTS / 4;
  static constexpr int W_OPS = (W_PER_WAVE + 63) / 64;  // DMA instructions per wave per stage
  static constexpr int H_OPS = (H_PER_WAVE + 63) / 64;
  static constexpr int OPS = W_OPS + H_OPS;
  static_assert(W_SLOTS % 4 == 0 && H_SLOTS % 4 == 0, "slots split evenly over the waves");
  static_assert(W_PER_WAVE % 64 == 0 || W_PER_WAVE < 64, "whole or partial DMA instructions");
  static_assert(H_PER_WAVE % 64 == 0 || H_PER_WAVE < 64, "whole or partial DMA instructions");
  static_assert(WCH >= 16, "the swizzle permutes 16 chunks");
  static_assert(BK * (F32 ? 4 : 2) == 64, "h rows hold four 16-byte chunks per stage");
};

template <class L, int KC, bool F32>
struct DmaKernel {
  using G = DmaGeom<L, F32>;
  using E = typename std::conditional<F32, float, uint16_t>::type;
  static constexpr int BV = L::BV, BH = L::BH, WV = L::WV, WH = L::WH, NWV = L::NWV;
  static constexpr int BK = G::BK;
  // per-tile extras (bias, shared-threshold keys), issued with a tile's first stage
  static constexpr int B_SLOTS = BV / 4, B_PER_WAVE = B_SLOTS / 4;  // float4 chunks
  static constexpr int T_SLOTS = BH / 4, T_PER_WAVE = T_SLOTS / 4;  // uint4 chunks
  static_assert(B_PER_WAVE >= 1 && B_PER_WAVE <= 64 && T_PER_WAVE >= 1 && T_PER_WAVE <= 64, "one extra op each");

  // Per-lane parts of the DMA source addresses, fixed for the whole kernel.
  struct Offs {
    int wr[G::W_OPS], wc[G::W_OPS];  // W row within stage, word offset within tile
    int hoff[G::H_OPS];              // h element offset (row * H + chunk)
    int trow;                        // row whose shared-threshold key this lane copies
  };

  __device__ __forceinline__ static void offsets(Offs& o, const K1Args& a, int h0) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int i = 0; i < G::W_OPS; ++i) {
      const int s = wave * G::W_PER_WAVE + i * 64 + lane;
      const int r = s / G::WCH, pc = s % G::WCH;
      o.wr[i] = r;
      o.wc[i] = (F32 ? pc : (pc ^ wswz(r))) * G::EPC;
    }
#pragma unroll
    for (int i = 0; i < G::H_OPS; ++i) {
      // slot s = row * 4 + physical chunk; logical chunk = physical ^ hswz(row)
      const int s = wave * G::H_PER_WAVE + i * 64 + lane;
      const int n = s >> 2, pc = s & 3;
      o.hoff[i] = min(h0 + n, a.N - 1) * a.H + (pc ^ hswz(n)) * G::EPC;  // rows >= N: computed, never written
    }
    o.trow = h0 + (wave * T_PER_WAVE + lane) * 4;  // 4 keys per 16 bytes; the key array is padded to whole row tiles
  }

  // Stage (v0, k0) into LDS stage buffer sb (W then h); a tile's first stage
  // also brings that tile's bias and shared-threshold keys into ep slot par.
  __device__ __forceinline__ static void issue(const K1Args& a, const Offs& o, uint32_t sb, int v0, int k0,
                                               uint32_t bias_lds, uint32_t tgk_lds) {
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const E* W = reinterpret_cast<const E*>(a.W) + (size_t)k0 * a.V;
    const E* h = reinterpret_cast<const E*>(a.h) + k0;
    const bool ragged = v0 + BV > a.V;
#pragma unroll
    for (int i = 0; i < G::W_OPS; ++i) {
      if (G::W_PER_WAVE >= 64 || lane < G::W_PER_WAVE) {
        int v = v0 + o.wc[i];
        if (ragged) v = min(v, a.V - G::EPC);  // words >= V are masked in the epilogue
        dma16(W + (size_t)o.wr[i] * a.V + v, sb + (wave * G::W_PER_WAVE + i * 64) * 16);
      }
    }
    const uint32_t hb = sb + G::W_SLOTS * 16;
#pragma unroll
    for (int i = 0; i < G::H_OPS; ++i) {
      if (G::H_PER_WAVE >= 64 || lane < G::H_PER_WAVE)
        dma16(h + o.hoff[i], hb + (wave * G::H_PER_WAVE + i * 64) * 16);
    }
    if (k0 == 0) {
      if (lane < B_PER_WAVE) {
        const int v = min(v0 + (wave * B_PER_WAVE + lane) * 4, a.V - 4);  // words >= V are masked
        dma16(a.b + v, bias_lds + wave * B_PER_WAVE * 16);
      }
      if (a.share && lane < T_PER_WAVE) dma16(a.gthr + o.trow, tgk_lds + wave * T_PER_WAVE * 16);
    }
  }

  __device__ __forceinline__ static void compute(f32x16 (&acc)[WV][WH], const uint16_t* Wb, const uint16_t* Hb) {
    if constexpr (F32) {
      compute_f32(acc, reinterpret_cast<const float*>(Wb), reinterpret_cast<const float*>(Hb));
      return;
    }
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wv = wave % NWV, wh = wave / NWV;
    const int g = lane >> 4, j = lane & 15;
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      bf16x8 af[WV], bf[WH];
      const int r0 = kk * 16 + 8 * (g >> 1) + (j >> 2);
#pragma unroll
      for (int vb = 0; vb < WV; ++vb) {
        const int colw = (wv * WV + vb) * 32 + 16 * (g & 1) + 4 * (j & 3);
        const int lc = colw >> 3, e = colw & 7;
        const int a0 = r0 * BV + ((lc ^ wswz(r0)) << 3) + e;
        const int a1 = a0 + 4 * BV;  // rows r0 + 4: same swizzle
        const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((KB_LDS s16x4*)(Wb + a0));
        const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((KB_LDS s16x4*)(Wb + a1));
        af[vb] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
      }
#pragma unroll
      for (int hb = 0; hb < WH; ++hb) {
        const int n = (wh * WH + hb) * 32 + (lane & 31);
        const int kc = kk * 2 + (lane >> 5);
        bf[hb] = *reinterpret_cast<const bf16x8*>(Hb + (n * 4 + (kc ^ hswz(n))) * 8);
      }
#pragma unroll
      for (int vb = 0; vb < WV; ++vb)
#pragma unroll
        for (int hb = 0; hb < WH; ++hb)
          acc[vb][hb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[vb], bf[hb], acc[vb][hb], 0, 0, 0);
    }
  }

  // float32: step 4 c + s (c < 2, s < 4) of the stage pairs, in lane half g,
  // state 8 g + 4 c + s: A (W, [state][word]) one float per lane, B (h)
  // element s of the lane's 16-byte chunk 2 g + c of its row
  __device__ __forceinline__ static void compute_f32(f32x16 (&acc)[WV][WH], const float* Wb, const float* Hb) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wv = wave % NWV, wh = wave / NWV;
    const int g = lane >> 5, col = lane & 31;
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      float4 hq[WH];
#pragma unroll
      for (int hb = 0; hb < WH; ++hb) {
        const int n = (wh * WH + hb) * 32 + col;
        hq[hb] = *reinterpret_cast<const float4*>(Hb + (n * 4 + ((2 * g + c) ^ hswz(n))) * 4);
      }
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const int kr = 8 * g + 4 * c + s;
        float af[WV];
#pragma unroll
        for (int vb = 0; vb < WV; ++vb) af[vb] = Wb[kr * BV + (wv * WV + vb) * 32 + col];
#pragma unroll
        for (int vb = 0; vb < WV; ++vb)
#pragma unroll
          for (int hb = 0; hb < WH; ++hb) {
            const float bv = s == 0 ? hq[hb].x : (s == 1 ? hq[hb].y : (s == 2 ? hq[hb].z : hq[hb].w));
            acc[vb][hb] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[vb], bv, acc[vb][hb], 0, 0, 0);
          }
      }
    }
  }
};

// Waves per SIMD the compiler must leave registers for: two for the 64-row x
// 128-word tile with k <= 8 (two workgroups per CU; the accumulators then sit
// in the architectural registers, at most 256 per lane in all), else one.
constexpr int dma_waves_per_eu(int bh, int bv, int kc) { return bh == 64 && bv == 128 && kc <= 8 ? 2 : 1; }

template <class L, int KC, bool F32>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(dma_waves_per_eu(L::BH, L::BV, KC))))
void k1_dma(K1Args a) {
  using D = DmaKernel<L, KC, F32>;
  using G = DmaGeom<L, F32>;
  constexpr int BV = L::BV, BH = L::BH, WV = L::WV, WH = L::WH, NWV = L::NWV;
  constexpr int WE = G::W_SLOTS * 8, HE = G::H_SLOTS * 8;  // 2-byte units per stage
  // one __shared__ object per stage: W, then h
  __shared__ __attribute__((aligned(16))) uint16_t S0[WE + HE], S1[WE + HE], S2[WE + HE], S3[WE + HE];
  __shared__ __attribute__((aligned(16))) SmemEpi<L> ep;
  static_assert(G::NS == 4, "four named stage buffers");
  // DMA accounting: every wave issues OPS instructions per stage, plus 2 with
  // a tile's first stage.  Waiting for "at most 2*OPS outstanding" therefore
  // always covers the oldest stage in flight (extra ops only make it stricter).

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int row_tile, split;
  k1_cell(a, blockIdx.x, row_tile, split);
  const int h0 = row_tile * BH;
  const int vt0 = split * a.tps;
  const int vt1 = min(vt0 + a.tps, a.n_vtiles);
  const int nk = a.H / G::BK;  // a multiple of 4: every tile starts on ring buffer 0
  const int total = (vt1 - vt0) * nk;
  const uint32_t sbuf[4] = {lds_addr(S0), lds_addr(S1), lds_addr(S2), lds_addr(S3)};

  Epilogue<L, KC> epi;
  epi.init(ep, a.k);
  typename D::Offs offs;
  D::offsets(offs, a, h0);

  // next stage to issue: tile start iv0 (tile index it), state offset ik0
  int iv0 = vt0 * BV, ik0 = 0, it = 0, issued = 0;
  auto issue_next = [&](int buf) {
    if (issued < total) {
      D::issue(a, offs, sbuf[buf], iv0, ik0, lds_addr(&ep.bias[it & 1][0]), lds_addr(&ep.tgk[it & 1][0]));
      ++issued;
      ik0 += G::BK;
      if (ik0 == a.H) {
        ik0 = 0;
        iv0 += BV;
        ++it;
      }
    }
  };
  issue_next(0);
  issue_next(1);
  issue_next(2);

  // stage g: wait for this thread's DMA of g (later stages may stay in flight),
  // barrier (all threads' data of g landed, stage g-1 consumed), refill the
  // buffer of g-1 with stage g+3, compute on g.
  auto wait_stage = [&](int g) {
    const int ahead = total - 1 - g;
    if (ahead >= 2)
      wait_vm<2 * G::OPS>();
    else if (ahead == 1)
      wait_vm<G::OPS>();
    else
      wait_vm<0>();
    lds_barrier();
  };

  int g = 0;
  for (int vt = vt0; vt < vt1; ++vt) {
    f32x16 acc[WV][WH];
#pragma unroll
    for (int vb = 0; vb < WV; ++vb)
#pragma unroll
      for (int hb = 0; hb < WH; ++hb)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[vb][hb][r] = 0.f;
    for (int kt = 0; kt < nk; kt += 4, g += 4) {
      wait_stage(g);
      issue_next(3);
      D::compute(acc, S0, S0 + WE);
      wait_stage(g + 1);
      issue_next(0);
      D::compute(acc, S1, S1 + WE);
      wait_stage(g + 2);
      issue_next(1);
      D::compute(acc, S2, S2 + WE);
      wait_stage(g + 3);
      issue_next(2);
      D::compute(acc, S3, S3 + WE);
    }
    // this tile's bias and keys landed with its first stage (waited for above)
    const int par = (vt - vt0) & 1;
    uint32_t tg[WH];
    {
      const int wh = wave / NWV, col = lane & 31;
#pragma unroll
      for (int hb = 0; hb < WH; ++hb) tg[hb] = a.share ? ep.tgk[par][(wh * WH + hb) * 32 + col] : 0u;
    }
    epi.tile(acc, ep, a, h0, vt * BV, vt == vt0, tg, ep.bias[par]);
  }
  epi.finish(ep, a, h0, split);
}

template <class L, bool F32 = false>
hipError_t launch_k1_dma_layout(int kc, dim3 grid, const K1Args& a, hipStream_t st) {
  const dim3 block(256);
  switch (kc) {
    case 4: k1_dma<L, 4, F32><<<grid, block, 0, st>>>(a); break;
    case 8: k1_dma<L, 8, F32><<<grid, block, 0, st>>>(a); break;
    case 12: k1_dma<L, 12, F32><<<grid, block, 0, st>>>(a); break;
    case 16: k1_dma<L, 16, F32><<<grid, block, 0, st>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace kb
