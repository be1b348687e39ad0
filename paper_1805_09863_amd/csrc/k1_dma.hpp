// K1, DMA variant: the fused output-layer projection for bf16 h and W with
// H % 32 == 0, V % 8 == 0 and 16-byte aligned operands (the production path).
//
// Same work split and epilogue as the register-staged kernel; the difference
// is how operands reach the matrix cores.  A ring of NS LDS stages (BK = 32
// of the state dimension each) is filled by the gfx950 global->LDS DMA
// (global_load_lds_dwordx4), so loads need no VGPRs and several stages are
// in flight while the MFMAs consume another:
//   * W keeps its V-contiguous layout in LDS; each 16-byte chunk of a row is
//     XOR-swizzled by the row index, and MFMA A-fragments (8 consecutive k
//     of one word) are built with the LDS transpose read ds_read_b64_tr_b16;
//   * h is stored chunk-major ([k/8][row][8]) so that B-fragments are
//     conflict-free 16-byte reads.
// Each stage has its own __shared__ array, which lets the compiler see that
// MFMA-side LDS reads never alias the DMA writes still in flight; the kernel
// waits on the vector-memory counter itself (s_waitcnt vmcnt).
#pragma once

#include "k1_common.hpp"

namespace kb {

#define KB_LDS __attribute__((address_space(3)))
typedef short s16x4 __attribute__((ext_vector_type(4)));

template <class L>
struct DmaGeom {
  static constexpr int BK = 32;                 // K per stage
  static constexpr int NS = 4;                  // stages in the ring
  static constexpr int WCH = L::BV / 8;         // 16-byte chunks per W row
  static constexpr int W_SLOTS = BK * WCH;      // 16-byte chunks of W per stage
  static constexpr int H_SLOTS = L::BH * BK / 8;
  static constexpr int W_PER_WAVE = W_SLOTS / 4;
  static constexpr int H_PER_WAVE = H_SLOTS / 4;
  static constexpr int W_OPS = (W_PER_WAVE + 63) / 64;  // DMA instructions per wave per stage
  static constexpr int H_OPS = (H_PER_WAVE + 63) / 64;
  static constexpr int OPS = W_OPS + H_OPS;
  static_assert(W_SLOTS % 4 == 0 && H_SLOTS % 4 == 0, "slots split evenly over the waves");
  static_assert(W_PER_WAVE % 64 == 0 || W_PER_WAVE < 64, "whole or partial DMA instructions");
  static_assert(H_PER_WAVE % 64 == 0 || H_PER_WAVE < 64, "whole or partial DMA instructions");
  static_assert(WCH >= 16, "the swizzle permutes 16 chunks");
};

// XOR swizzle of the 16-byte chunks of W row r: rows r..r+3 read together by
// one transpose read land on distinct banks.
__device__ __forceinline__ int wswz(int r) { return 4 * (r & 3) + 2 * ((r >> 1) & 1); }

// s_waitcnt vmcnt(n) with expcnt / lgkmcnt left alone (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

template <class L, int KC>
struct DmaKernel {
  using G = DmaGeom<L>;
  static constexpr int BV = L::BV, BH = L::BH, WV = L::WV, WH = L::WH, NWV = L::NWV;
  static constexpr int BK = G::BK;

  // one DMA wave-instruction: 64 consecutive 16-byte LDS slots from base
  __device__ __forceinline__ static void dma16(const void* g, KB_LDS void* lds_base) {
    __builtin_amdgcn_global_load_lds(g, lds_base, 16, 0, 0);
  }

  __device__ __forceinline__ static void issue(const K1Args& a, uint16_t* Wb, uint16_t* Hb, int h0, int v0,
                                               int k0) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const uint16_t* W = reinterpret_cast<const uint16_t*>(a.W);
    const uint16_t* h = reinterpret_cast<const uint16_t*>(a.h);
#pragma unroll
    for (int i = 0; i < G::W_OPS; ++i) {
      const int slot0 = wave * G::W_PER_WAVE + i * 64;
      if (G::W_PER_WAVE >= 64 || lane < G::W_PER_WAVE) {
        const int s = slot0 + lane;
        const int r = s / G::WCH, pc = s % G::WCH;
        const int lc = pc ^ wswz(r);
        const int v = min(v0 + lc * 8, a.V - 8);  // words >= V are masked in the epilogue
        dma16(W + (size_t)(k0 + r) * a.V + v, (KB_LDS void*)(Wb + slot0 * 8));
      }
    }
#pragma unroll
    for (int i = 0; i < G::H_OPS; ++i) {
      const int slot0 = wave * G::H_PER_WAVE + i * 64;
      if (G::H_PER_WAVE >= 64 || lane < G::H_PER_WAVE) {
        const int s = slot0 + lane;
        const int kc = s / BH, n = s % BH;
        const int row = min(h0 + n, a.N - 1);  // rows >= N are computed and never written
        dma16(h + (size_t)row * a.H + k0 + kc * 8, (KB_LDS void*)(Hb + slot0 * 8));
      }
    }
  }

  __device__ __forceinline__ static void compute(f32x16 (&acc)[WV][WH], const uint16_t* Wb, const uint16_t* Hb) {
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
        const short t8[8] = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        __builtin_memcpy(&af[vb], t8, 16);
      }
#pragma unroll
      for (int hb = 0; hb < WH; ++hb)
        bf[hb] = *reinterpret_cast<const bf16x8*>(
            Hb + ((kk * 2 + (lane >> 5)) * BH + (wh * WH + hb) * 32 + (lane & 31)) * 8);
#pragma unroll
      for (int vb = 0; vb < WV; ++vb)
#pragma unroll
        for (int hb = 0; hb < WH; ++hb)
          acc[vb][hb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[vb], bf[hb], acc[vb][hb], 0, 0, 0);
    }
  }
};

template <class L, int KC>
__global__ __launch_bounds__(256) void k1_dma(K1Args a) {
  using D = DmaKernel<L, KC>;
  using G = DmaGeom<L>;
  constexpr int BV = L::BV, BH = L::BH, WV = L::WV, WH = L::WH;
  constexpr int WE = G::W_SLOTS * 8, HE = G::H_SLOTS * 8;  // bf16 elements per stage
  __shared__ __attribute__((aligned(16))) uint16_t W0[WE], W1[WE], W2[WE], W3[WE];
  __shared__ __attribute__((aligned(16))) uint16_t H0[HE], H1[HE], H2[HE], H3[HE];
  __shared__ SmemEpi<L> ep;
  static_assert(G::NS == 4, "four named stage buffers");

  const int tid = threadIdx.x;
  const int split = blockIdx.x;
  const int h0 = blockIdx.y * BH;
  const int vt0 = split * a.tps;
  const int vt1 = min(vt0 + a.tps, a.n_vtiles);
  const int nk = a.H / G::BK;
  const int total = (vt1 - vt0) * nk;

  Epilogue<L, KC> epi;
  epi.init(ep, a.k);

  // stage g covers tile vt0 + g / nk, state rows (g % nk) * BK ..
  auto issue_g = [&](int g, uint16_t* Wb, uint16_t* Hb) {
    const int t = g / nk, kt = g - t * nk;
    D::issue(a, Wb, Hb, h0, (vt0 + t) * BV, kt * G::BK);
  };
  issue_g(0, W0, H0);
  if (total > 1) issue_g(1, W1, H1);
  if (total > 2) issue_g(2, W2, H2);

  float tg[WH];
  epi.load_shared_thr(a, h0, tg);
  f32x16 acc[WV][WH];
#pragma unroll
  for (int vb = 0; vb < WV; ++vb)
#pragma unroll
    for (int hb = 0; hb < WH; ++hb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[vb][hb][r] = 0.f;

  int kt = 0, vt = vt0;
  for (int g = 0; g < total; ++g) {
    // wait for this thread's DMA of stage g (later issued stages may stay in flight)
    const int ahead = total - 1 - g;
    if (ahead >= 2)
      wait_vm<2 * G::OPS>();
    else if (ahead == 1)
      wait_vm<G::OPS>();
    else
      wait_vm<0>();
    lds_barrier();  // every thread's stage-g data landed; stage g-1 fully consumed
    if (kt == 0)
      for (int i = tid; i < BV; i += 256) ep.bias[i] = (vt * BV + i < a.V) ? a.b[vt * BV + i] : 0.f;
    switch (g & 3) {
      case 0:
        if (g + 3 < total) issue_g(g + 3, W3, H3);
        D::compute(acc, W0, H0);
        break;
      case 1:
        if (g + 3 < total) issue_g(g + 3, W0, H0);
        D::compute(acc, W1, H1);
        break;
      case 2:
        if (g + 3 < total) issue_g(g + 3, W1, H1);
        D::compute(acc, W2, H2);
        break;
      default:
        if (g + 3 < total) issue_g(g + 3, W2, H2);
        D::compute(acc, W3, H3);
        break;
    }
    if (++kt == nk) {
      lds_barrier();  // bias visible
      epi.tile(acc, ep, a, h0, vt * BV, vt == vt0, tg);
      kt = 0;
      ++vt;
      if (vt < vt1) epi.load_shared_thr(a, h0, tg);
#pragma unroll
      for (int vb = 0; vb < WV; ++vb)
#pragma unroll
        for (int hb = 0; hb < WH; ++hb)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[vb][hb][r] = 0.f;
    }
  }
  epi.finish(ep, a, h0, split);
}

template <class L>
hipError_t launch_k1_dma_layout(int kc, dim3 grid, const K1Args& a, hipStream_t st) {
  const dim3 block(256);
  switch (kc) {
    case 4: k1_dma<L, 4><<<grid, block, 0, st>>>(a); break;
    case 8: k1_dma<L, 8><<<grid, block, 0, st>>>(a); break;
    case 12: k1_dma<L, 12><<<grid, block, 0, st>>>(a); break;
    case 16: k1_dma<L, 16><<<grid, block, 0, st>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace kb
