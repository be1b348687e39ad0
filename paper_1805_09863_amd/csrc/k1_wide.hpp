// K1, wide variant: the fused output-layer projection for many live rows
// (bf16 h and W, H % 128 == 0, V % 8 == 0, 16-byte aligned operands).
//
// Tile: 256 words x 256 hypothesis rows per workgroup of four waves; wave
// (wv, wh) owns words [128 wv, 128 wv + 128) and rows [128 wh, 128 wh + 128)
// as 4 x 4 accumulators of v_mfma_f32_32x32x16_bf16 (256 registers, kept in
// the accumulation registers).  A square tile moves 1 KB of operands per 16
// states for 131k flops, half the operand bytes per flop of a 128 x 256 tile,
// which keeps the global->LDS stream well below what a CU can sustain.
//
// Operands reach LDS through a ring of four stages (32 states each) filled by
// the gfx950 global->LDS DMA, with a wave-uniform base in SGPRs and fixed
// per-lane offsets, so issuing a stage costs eight instructions per wave.
// Layouts and swizzles are those of the narrow DMA kernel: W stays
// V-contiguous (A-fragments via the LDS transpose read), h rows are
// row-major 64-byte slices per stage.
//
// Per stage the wave reads the second half of its fragments, runs the first
// half's 16 MFMAs, waits for the next stage and passes the only barrier of
// the stage, refills the buffer it just finished with the stage four ahead,
// reads the next stage's first fragments and runs the second half's MFMAs.
// LDS reads therefore always overlap MFMAs, and no wait drains the ring.
//
// Epilogue per tile (the accumulators start at the bias, so Algorithm 3's
// AddBias costs nothing; words >= V start at -inf and drop out everywhere):
//   * per row of the lane: tile max (3-input max tree), then the running
//     (max, sum) with one rescale per tile (Algorithm 4's identity);
//   * rows whose tile max reaches max(local k-th best, shared threshold)
//     append their candidates to a per-row LDS list; the owner thread of the
//     row inserts them into its sorted k-list (registers) and raises the
//     thresholds.  Ties are kept by the filter and settled by word index.
#pragma once

#include <type_traits>

#include "k1_common.hpp"

namespace kb {

__device__ __forceinline__ float fmax3(float a, float b, float c) { return fmaxf(fmaxf(a, b), c); }

struct WideGeom {
  static constexpr int BV = 256, BH = 256, BK = 32;
  static constexpr int WE = BK * BV;  // bf16 elements of W per stage
  static constexpr int HE = BH * BK;  // bf16 elements of h per stage
  static constexpr int OPS = 8;       // DMA instructions per wave per stage
  static constexpr int CAP = 12;      // candidate slots per row per round
  static constexpr int DONE = 64;     // "no pending candidates" position
};

struct alignas(16) WideEpi {
  float bias[2][WideGeom::BV];    // bias of the current / next tile (DMA)
  uint32_t tgk[2][WideGeom::BH];  // shared-threshold keys of the current / next tile (DMA)
  float thr[WideGeom::BH];        // row's local threshold: its k-th best so far, or the seed
  int cnt[WideGeom::BH];          // candidates appended to the row this round
  int flag[4];                    // "a lane could not append" of this and the next round
  union {
    int2 cand[WideGeom::BH][WideGeom::CAP];  // (score bits, word) appended this round
    float red[WideGeom::BH][8];              // seeds, then the per-holder statistics
  } u;
};

// One global->LDS DMA wave-instruction with a wave-uniform base (SGPR pair)
// and a per-lane 32-bit byte offset: lane i copies 16 bytes from
// base + voff to LDS byte lds_base + 16 i.
__device__ __forceinline__ void dma16_so(uint32_t voff, const void* sbase, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(sbase),
               "s"(lds_base)
               : "m0");
}

// Marks an accumulator block as redefined in place (it stays in the
// accumulation registers).  Used at the start of each row's epilogue work so
// that the compiler copies only that row's 64 scores into VGPRs, and copies
// them again in each candidate round instead of keeping all 256 alive.
__device__ __forceinline__ void opaque(f32x16& x) { asm volatile("" : "+a"(x)); }

// A row's results "used" at a point that, being volatile, stays ordered
// before the next row's opaque(): together they keep the compiler from
// interleaving consecutive rows (which would hold several rows' 64 scores in
// VGPRs at once).
__device__ __forceinline__ void done(float x) { asm volatile("" ::"v"(x)); }
__device__ __forceinline__ void done(int x) { asm volatile("" ::"v"(x)); }

__device__ __forceinline__ float max4(const f32x16& x, int q) {
  return fmaxf(fmax3(x[4 * q], x[4 * q + 1], x[4 * q + 2]), x[4 * q + 3]);
}

template <int KC>
__global__ __launch_bounds__(256, 1) void k1_wide(K1Args a) {
  using G = WideGeom;
  constexpr int BV = G::BV, BH = G::BH, BK = G::BK, WE = G::WE, HE = G::HE;
  __shared__ __attribute__((aligned(16))) uint16_t S0[WE + HE], S1[WE + HE], S2[WE + HE], S3[WE + HE];
  __shared__ WideEpi ep;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wv = wave & 1, wh = wave >> 1;
  const int half = lane >> 5, col = lane & 31;
  const int holder = wv * 2 + half;  // which of the row's four holders this lane is
  const int k = a.k;

  int row_tile, split;
  k1_cell(a, blockIdx.x, row_tile, split);
  const int h0 = row_tile * BH;
  const int vt0 = split * a.tps;
  const int vt1 = min(vt0 + a.tps, a.n_vtiles);
  const int nk = a.H / BK;  // a multiple of 4: every tile starts on ring buffer 0
  const int total = (vt1 - vt0) * nk;

  // ---- per-lane DMA byte offsets (fixed for the whole kernel)
  // W slot s = 256 wave + 64 i + lane: stage row r = s / 32, physical chunk
  // s % 32 holding logical chunk (s % 32) ^ wswz(r).
  // h slot s: row n = s / 4, physical chunk s % 4 holding chunk (s % 4) ^ hswz(n).
  uint32_t woff[4], hoff[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = wave * 8 + i * 2 + half;
    woff[i] = (uint32_t)r * (uint32_t)a.V * 2u + (uint32_t)((col ^ wswz(r)) * 16);
    const int n = wave * 64 + i * 16 + (lane >> 2);
    hoff[i] = (uint32_t)min(h0 + n, a.N - 1) * (uint32_t)a.H * 2u + (uint32_t)(((lane & 3) ^ hswz(n)) * 16);
  }

  auto issue = [&](uint16_t* buf, int v0, int k0, int par) {
    const uint32_t sb = lds_addr(buf);
    const char* Wp = reinterpret_cast<const char*>(a.W) + ((size_t)k0 * a.V + v0) * 2;
    const char* Hp = reinterpret_cast<const char*>(a.h) + (size_t)k0 * 2;
    if (v0 + BV <= a.V) {
#pragma unroll
      for (int i = 0; i < 4; ++i) dma16_so(woff[i], Wp, sb + (wave * 256 + i * 64) * 16);
    } else {  // last, ragged tile: words >= V read word V - 8.. instead (they start at -inf)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = wave * 8 + i * 2 + half;
        const int w = min(v0 + (col ^ wswz(r)) * 8, a.V - 8) - v0;
        dma16_so((uint32_t)r * (uint32_t)a.V * 2u + (uint32_t)w * 2u, Wp, sb + (wave * 256 + i * 64) * 16);
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) dma16_so(hoff[i], Hp, sb + WE * 2 + (wave * 256 + i * 64) * 16);
    if (k0 == 0) {  // the tile's bias and shared-threshold keys ride with its first stage
      if (wave == 0) {
        dma16(a.b + min(v0 + lane * 4, a.V - 4), lds_addr(&ep.bias[par][0]));
      } else if (wave == 1) {
        dma16(a.gthr + h0 + lane * 4, lds_addr(&ep.tgk[par][0]));
      }
    }
  };

  int iv0 = vt0 * BV, ik0 = 0, it = 0, issued = 0;
  auto issue_next = [&](uint16_t* buf) {
    if (issued < total) {
      issue(buf, iv0, ik0, it & 1);
      ++issued;
      ik0 += BK;
      if (ik0 == a.H) {
        ik0 = 0;
        iv0 += BV;
        ++it;
      }
    }
  };

  // ---- MFMA fragments of one 16-state step (kk) of a stage.  Per-lane byte
  // offsets within a stage buffer: A (W^T) fragments of block vb at kk = 0
  // (kk adds 16 rows, which leaves the swizzle unchanged); B (h) fragments of
  // block 0 at each kk (blocks are 32 rows = 2 KB apart, same swizzle).
  uint32_t aoff[4], boff[2];
  {
    const int g = lane >> 4, j = lane & 15;
    const int r0 = 8 * (g >> 1) + (j >> 2);
#pragma unroll
    for (int vb = 0; vb < 4; ++vb) {
      const int colw = wv * 128 + vb * 32 + 16 * (g & 1) + 4 * (j & 3);
      aoff[vb] = (uint32_t)(r0 * BV + (((colw >> 3) ^ wswz(r0)) << 3) + (colw & 7)) * 2u;
    }
    const int n = wh * 128 + col;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) boff[kk] = (uint32_t)(WE + n * 32 + (((kk * 2 + half) ^ hswz(n)) * 8)) * 2u;
  }
  auto load_frags = [&](const uint16_t* buf, int kk, bf16x8(&fa)[4], bf16x8(&fb)[4]) {
    const KB_LDS char* base = (const KB_LDS char*)(const KB_LDS void*)buf;
#pragma unroll
    for (int vb = 0; vb < 4; ++vb) {
      const KB_LDS char* p = base + aoff[vb] + kk * 16 * BV * 2;
      const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((KB_LDS s16x4*)p);
      const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((KB_LDS s16x4*)(p + 4 * BV * 2));
      const short t8[8] = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
      __builtin_memcpy(&fa[vb], t8, 16);
    }
#pragma unroll
    for (int hb = 0; hb < 4; ++hb) fb[hb] = *(const KB_LDS bf16x8*)(base + boff[kk] + hb * 2048);
  };

  f32x16 acc[4][4];
  auto mfma16 = [&](const bf16x8(&fa)[4], const bf16x8(&fb)[4]) {
#pragma unroll
    for (int vb = 0; vb < 4; ++vb)
#pragma unroll
      for (int hb = 0; hb < 4; ++hb)
        acc[vb][hb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[vb], fb[hb], acc[vb][hb], 0, 0, 0);
  };

  // ---- accumulators start at the tile's bias; words >= V at -inf
  auto init_acc = [&](int vt) {
    const int par = (vt - vt0) & 1;
    const int v0 = vt * BV;
    const bool ragged = v0 + BV > a.V;
    // word of (vb, i, j) is valid iff vb * 32 + 8 i + j < lim
    const int lim = a.V - v0 - wv * 128 - 4 * half;
#pragma unroll
    for (int vb = 0; vb < 4; ++vb) {
      f32x16 bv;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int wl = wv * 128 + vb * 32 + 8 * i + 4 * half;
        const float4 bb = *reinterpret_cast<const float4*>(&ep.bias[par][wl]);
        bv[4 * i + 0] = bb.x;
        bv[4 * i + 1] = bb.y;
        bv[4 * i + 2] = bb.z;
        bv[4 * i + 3] = bb.w;
        if (ragged) {
#pragma unroll
          for (int j = 0; j < 4; ++j)
            if (vb * 32 + 8 * i + j >= lim) bv[4 * i + j] = -INFINITY;
        }
      }
#pragma unroll
      for (int hb = 0; hb < 4; ++hb) {
        acc[vb][hb] = bv;
        opaque(acc[vb][hb]);  // written straight into the accumulation registers
      }
    }
  };

  // ---- epilogue state
  float st_m[4], st_s[4];  // running (max, sum of exp(x - max)) of the lane's rows
  float lval[KC];          // owner (row = tid): sorted k best of the split so far
  int lidx[KC];
  float published = kNoThr;
#pragma unroll
  for (int hb = 0; hb < 4; ++hb) {
    st_m[hb] = kStatInit;
    st_s[hb] = 0.f;
  }
  list_init<KC>(lval, lidx, k);
  ep.thr[tid] = kNoThr;
  ep.cnt[tid] = 0;
  if (tid < 4) ep.flag[tid] = 0;

  auto publish = [&](float v) {
    if (h0 + tid < a.N && v > published) {
      atomicMax(&a.gthr[h0 + tid], f2key(v));
      published = v;
    }
  };

  auto epilogue = [&](int vt) {
    const int par = (vt - vt0) & 1;
    const int v0 = vt * BV;
    float tmax[4];
    // statistics (Algorithm 4, one rescale per tile)
#pragma unroll
    for (int hb = 0; hb < 4; ++hb) {
#pragma unroll
      for (int vb = 0; vb < 4; ++vb) opaque(acc[vb][hb]);
      float m0 = fmax3(acc[0][hb][0], acc[0][hb][1], acc[0][hb][2]);
      float m1 = fmax3(acc[0][hb][3], acc[0][hb][4], acc[0][hb][5]);
#pragma unroll
      for (int vb = 0; vb < 4; ++vb)
#pragma unroll
        for (int r = (vb == 0 ? 6 : 0); r < 16; r += 4) {
          m0 = fmax3(m0, acc[vb][hb][r], acc[vb][hb][r + 1]);
          m1 = fmax3(m1, acc[vb][hb][r + 2], acc[vb][hb][r + 3]);
        }
      const float mx = fmaxf(m0, m1);
      tmax[hb] = mx;
      const float mnew = fmaxf(st_m[hb], mx);
      const float ml2 = mnew * kL2E;
      float s0 = st_s[hb] * exp2_fast((st_m[hb] - mnew) * kL2E), s1 = 0.f;
#pragma unroll
      for (int vb = 0; vb < 4; ++vb)
#pragma unroll
        for (int r = 0; r < 16; r += 2) {
          s0 += exp2_fast(fmaf(acc[vb][hb][r], kL2E, -ml2));
          s1 += exp2_fast(fmaf(acc[vb][hb][r + 1], kL2E, -ml2));
        }
      st_s[hb] = s0 + s1;
      st_m[hb] = mnew;
      done(st_s[hb]);
      done(mx);
    }

    // first tile of the split: seed each row's threshold.  Every holder finds
    // the j-th largest of its 16 quad maxima (j = ceil(k / 4)); the row then
    // has at least 4 j >= k distinct scores >= the smallest of the four.
    if (vt == vt0) {
      const int jj = (k + 3) >> 2;
#pragma unroll
      for (int hb = 0; hb < 4; ++hb) {
#pragma unroll
        for (int vb = 0; vb < 4; ++vb) opaque(acc[vb][hb]);
        float sv[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) sv[j] = (j < 4 - jj) ? INFINITY : -INFINITY;
#pragma unroll
        for (int vb = 0; vb < 4; ++vb)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            float x = max4(acc[vb][hb], q);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const float hi = fmaxf(sv[j], x);
              x = fminf(sv[j], x);
              sv[j] = hi;
            }
          }
        ep.u.red[wh * 128 + hb * 32 + col][holder] = sv[3];
        done(sv[3]);
      }
      lds_barrier();
      {
        const float seed = fminf(fminf(ep.u.red[tid][0], ep.u.red[tid][1]), fminf(ep.u.red[tid][2], ep.u.red[tid][3]));
        if (seed > ep.thr[tid]) {
          ep.thr[tid] = seed;
          publish(seed);
        }
      }
      lds_barrier();
    }

    // candidate rounds: a lane appends, in position order, every score >= the
    // row's threshold; if the row's list is full it stops at that position and
    // resumes there in the next round, against the raised threshold
    int resume[4];
#pragma unroll
    for (int hb = 0; hb < 4; ++hb) {
      const int rl = wh * 128 + hb * 32 + col;
      const float t = fmaxf(ep.thr[rl], key2f(ep.tgk[par][rl]));
      resume[hb] = tmax[hb] >= t ? 0 : G::DONE;
    }
    for (int round = 0;; ++round) {
      int ovf = 0;
#pragma unroll
      for (int hb = 0; hb < 4; ++hb) {
        if (resume[hb] < G::DONE) {
#pragma unroll
          for (int vb = 0; vb < 4; ++vb) opaque(acc[vb][hb]);
          const int rl = wh * 128 + hb * 32 + col;
          const float t = fmaxf(ep.thr[rl], key2f(ep.tgk[par][rl]));
          const int rs = resume[hb];
          // word of position (vb, q, j) = wbase + 32 vb + 8 q + j; opaque so that
          // the 64 words are formed on demand, not hoisted out of the loop
          int wbase = v0 + wv * 128 + 4 * half;
          asm volatile("" : "+v"(wbase));
          int newres = G::DONE;
#pragma unroll
          for (int vb = 0; vb < 4; ++vb)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              if (max4(acc[vb][hb], q) >= t && vb * 16 + 4 * q + 3 >= rs && newres == G::DONE) {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                  const int pos = vb * 16 + 4 * q + j;
                  const float x = acc[vb][hb][4 * q + j];
                  if (x >= t && pos >= rs && newres == G::DONE) {
                    const int slot = atomicAdd(&ep.cnt[rl], 1);
                    if (slot < G::CAP)
                      ep.u.cand[rl][slot] = make_int2(__float_as_int(x), wbase + vb * 32 + 8 * q + j);
                    else
                      newres = pos;
                  }
                }
              }
            }
          resume[hb] = newres;
          ovf |= newres != G::DONE;
          done(newres);
        }
      }
      if (ovf) ep.flag[round & 1] = 1;
      lds_barrier();
      if (tid == 0) ep.flag[(round + 1) & 1] = 0;  // read only after the next barrier
      {
        const int c = min(ep.cnt[tid], G::CAP);
        for (int i = 0; i < c; ++i) {
          const int2 e = ep.u.cand[tid][i];
          const float cv = __int_as_float(e.x);
          if (better(cv, e.y, lval[KC - 1], lidx[KC - 1])) list_insert<KC>(lval, lidx, cv, e.y);
        }
        ep.cnt[tid] = 0;
        if (lval[KC - 1] > ep.thr[tid]) {
          ep.thr[tid] = lval[KC - 1];
          publish(lval[KC - 1]);
        }
      }
      lds_barrier();
      if (ep.flag[round & 1] == 0) break;
    }
  };

  // ---- the stage pipeline
  uint16_t* const bufs[4] = {S0, S1, S2, S3};
  bf16x8 fa0[4], fb0[4], fa1[4], fb1[4];

  issue_next(S0);
  issue_next(S1);
  issue_next(S2);
  issue_next(S3);
  // stage 0 landed: at most the three later stages outstanding
  if (total >= 4)
    wait_vm<3 * G::OPS>();
  else if (total == 3)
    wait_vm<2 * G::OPS>();
  else if (total == 2)
    wait_vm<G::OPS>();
  else
    wait_vm<0>();
  lds_barrier();
  init_acc(vt0);
  load_frags(S0, 0, fa0, fb0);

  int g = 0;
  auto body = [&](auto bc) {
    constexpr int b = decltype(bc)::value;
    uint16_t* const cur = bufs[b];
    uint16_t* const nxt = bufs[(b + 1) & 3];
    load_frags(cur, 1, fa1, fb1);
    __builtin_amdgcn_sched_barrier(0);
    mfma16(fa0, fb0);
    __builtin_amdgcn_sched_barrier(0);
    if (g + 1 < total) {
      const int ahead = total - 2 - g;  // stages issued after g + 1
      if (ahead >= 2)
        wait_vm<2 * G::OPS>();
      else if (ahead == 1)
        wait_vm<G::OPS>();
      else
        wait_vm<0>();
      lds_barrier();  // stage g + 1 landed everywhere; every wave is done with buffer b
      issue_next(cur);
      load_frags(nxt, 0, fa0, fb0);
    }
    __builtin_amdgcn_sched_barrier(0);
    mfma16(fa1, fb1);
    __builtin_amdgcn_sched_barrier(0);
    ++g;
  };

  for (int vt = vt0; vt < vt1; ++vt) {
    for (int kt = 0; kt < nk; kt += 4) {
      body(std::integral_constant<int, 0>{});
      body(std::integral_constant<int, 1>{});
      body(std::integral_constant<int, 2>{});
      body(std::integral_constant<int, 3>{});
    }
    epilogue(vt);
    if (vt + 1 < vt1) init_acc(vt + 1);
  }

  // ---- this split's partial of every row: merge the four holders' statistics
#pragma unroll
  for (int hb = 0; hb < 4; ++hb) {
    const int rl = wh * 128 + hb * 32 + col;
    ep.u.red[rl][2 * holder + 0] = st_m[hb];
    ep.u.red[rl][2 * holder + 1] = st_s[hb];
  }
  lds_barrier();
  if (h0 + tid < a.N) {
    float M = kStatInit;
#pragma unroll
    for (int i = 0; i < 4; ++i) M = fmaxf(M, ep.u.red[tid][2 * i]);
    float S = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) S += ep.u.red[tid][2 * i + 1] * exp2_fast((ep.u.red[tid][2 * i] - M) * kL2E);
    const size_t row = (size_t)split * a.N + h0 + tid;
    a.stats[row] = make_float2(M, S);
#pragma unroll
    for (int j = 0; j < KC; ++j)
      if (j >= KC - k) a.lists[row * k + (j - (KC - k))] = make_int2(__float_as_int(lval[j]), lidx[j]);
  }
}

template <int KC>
hipError_t launch_k1_wide_kc(dim3 grid, const K1Args& a, hipStream_t st) {
  k1_wide<KC><<<grid, dim3(256), 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace kb
