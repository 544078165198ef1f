// Integerised path kernels (Sec. 4.5; Supp. B.4, Alg. 1) for gfx950.
//
// CDNA4 has no int16 matrix instruction, so every int16 x int16 -> int32
// contraction is done exactly on the int8 MFMA: activations split as
// x = 256 xh + xl' + 128 (xh = x >> 8, xl' = (x & 255) - 128) and weights as
// balanced digits w = 256 wh + wl, giving
//   sum x w = 65536 sum xh wh + 256 (sum xh wl + sum xl' wh) + sum xl' wl + 128 sum w.
// Each partial sum fits int32 for K <= 1024; the final combination wraps
// modulo 2^32 exactly like an int32 accumulator, so the result equals the
// exact sum whenever that sum fits int32 (the paper's accumulator contract).
// The 128 sum w term and the bias term 512 b_i are pre-added per output
// channel ("corr").  Every conv then rescales with round-half-to-even of
// a / 8192 and saturates to int16.
#include "common.hpp"
#include "internal.hpp"

#include <cstring>

namespace nc {

// clip(RHE(a / 8192)) for any int32 a.  |a| >= 2^28 saturates either way, so a
// is first clamped to +-2^28; then the round-half-even bias can be added
// without overflow: RHE(a / 2^s) = (a + 2^(s-1) - 1 + ((a >> s) & 1)) >> s.
__device__ __forceinline__ int rescale13(int a) {
  const int ac = min(max(a, -(1 << 28)), 1 << 28);
  return clip16((ac + 4095 + ((ac >> 13) & 1)) >> 13);
}

__device__ __forceinline__ uint32_t pack2(int lo, int hi) {
  return ((uint32_t)lo & 0xFFFFu) | ((uint32_t)hi << 16);
}

// ---------------------------------------------------------------- pointwise
// Same tiling and LDS pipeline as the fp16 pointwise kernel: 8 waves per tile
// of 128 output pixels, K consumed 64 at a time through three LDS stages.  A
// stage holds the activation slice (int16, or the fp16 frame for the patch
// embed, converted with x_i = round(512 x) when the operand is read) and, per
// 32-row tile, four int8 fragments: hi digits for k-steps 0 and 1, then lo
// digits for k-steps 0 and 1 (32 contraction indices each).
struct PwSmemI {
  static constexpr int ACT = 128 * 128;
};
template <int NT>
struct PwSmemIN {
  static constexpr int WGT = NT / 32 * 4 * 1024;
  static constexpr int STAGE = PwSmemI::ACT + WGT;
  static constexpr int DMA_PER_WAVE = (PwSmemI::ACT / 1024 + WGT / 1024) / 8;
};

template <int LOADER>
__device__ __forceinline__ const char* pwi_act_src(const PwArgs& a, int gp, int kc, int v) {
  const int k = 64 * kc + 8 * v;
  if constexpr (LOADER == LD_NHWC) {
    if (k < a.C0) return (const char*)((const int16_t*)a.src0 + (size_t)gp * a.C0 + k);
    return (const char*)((const int16_t*)a.src1 + (size_t)gp * a.C1 + (k - a.C0));
  } else if constexpr (LOADER == LD_FRAME) {
    const int py = gp / a.w8, px = gp - py * a.w8;
    return (const char*)((const f16*)a.src0 + (size_t)kc * a.H * a.W + (size_t)(8 * py + v) * a.W + 8 * px);
  } else {
    const int w16 = a.w8 >> 1;
    const int Y = gp / w16, X = gp - Y * w16;
    const int tap = k / a.Csrc, c = k - tap * a.Csrc;
    const int pix = (2 * Y + (tap >> 1)) * a.w8 + 2 * X + (tap & 1);
    return (const char*)((const int16_t*)a.src0 + (size_t)pix * a.Csrc + c);
  }
}

template <int NT, int LOADER>
__device__ __forceinline__ void pwi_issue(const PwArgs& a, int tile, int n0, int kc, char* stage, int wave, int lane) {
  constexpr int ACT_INSTR = PwSmemI::ACT / 1024;
#pragma unroll
  for (int i = 0; i < ACT_INSTR / 8; ++i) {
    const int ins = wave + 8 * i;
    const int slot = ins * 64 + lane;
    const int px = slot >> 3, v = (slot & 7) ^ (px & 7);
    const int gp = min(tile * 128 + px, a.P - 1);
    dma16(pwi_act_src<LOADER>(a, gp, kc, v), stage + ins * 1024);
  }
  const int ks = a.K / 32;
#pragma unroll
  for (int i = 0; i < PwSmemIN<NT>::WGT / 1024 / 8; ++i) {
    const int f = wave + 8 * i;  // row tile f / 4; f % 4: hi k0, hi k1, lo k0, lo k1
    const int mt = n0 / 32 + (f >> 2), sk = 2 * kc + (f & 1);
    const char* plane = (f & 2) ? (const char*)a.wfrag_lo : (const char*)a.wfrag;
    dma16(plane + (((size_t)mt * ks + sk) * 64 + lane) * 16, stage + PwSmemI::ACT + f * 1024);
  }
}

template <int NT, int LOADER>
__device__ __forceinline__ void pwi_compute(const char* stage, int pg, int hf, int lane, intx16 (*acc)[3]) {
  constexpr int RT = NT / 64;
  const int pl = pg * 32 + (lane & 31), h = lane >> 5;
  intx4 bh[2], bl[2];
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
    // contraction indices 32 ks + 16 h .. +15 = vectors 4 ks + 2 h and + 1
    const int v0 = 4 * ks + 2 * h;
    uint32_t d[8];
    if constexpr (LOADER == LD_FRAME) {
      const half8 x0 = *(const half8*)(stage + pl * 128 + ((v0 ^ (pl & 7)) << 4));
      const half8 x1 = *(const half8*)(stage + pl * 128 + (((v0 + 1) ^ (pl & 7)) << 4));
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        d[e] = pack2(clip16((int)rintf((float)x0[2 * e] * 512.f)), clip16((int)rintf((float)x0[2 * e + 1] * 512.f)));
        d[4 + e] = pack2(clip16((int)rintf((float)x1[2 * e] * 512.f)), clip16((int)rintf((float)x1[2 * e + 1] * 512.f)));
      }
    } else {
      const intx4 q0 = *(const intx4*)(stage + pl * 128 + ((v0 ^ (pl & 7)) << 4));
      const intx4 q1 = *(const intx4*)(stage + pl * 128 + (((v0 + 1) ^ (pl & 7)) << 4));
#pragma unroll
      for (int e = 0; e < 4; ++e) { d[e] = (uint32_t)q0[e]; d[4 + e] = (uint32_t)q1[e]; }
    }
    split16(d, bh[ks], bl[ks]);
  }
#pragma unroll
  for (int t = 0; t < RT; ++t) {
    const char* wt = stage + PwSmemI::ACT + (hf * RT + t) * 4 * 1024 + lane * 16;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const intx4 wh = *(const intx4*)(wt + ks * 1024), wl = *(const intx4*)(wt + (2 + ks) * 1024);
      acc[t][0] = mfma_i8(wh, bh[ks], acc[t][0]);
      acc[t][1] = mfma_i8(wh, bl[ks], acc[t][1]);
      acc[t][1] = mfma_i8(wl, bh[ks], acc[t][1]);
      acc[t][2] = mfma_i8(wl, bl[ks], acc[t][2]);
    }
  }
}

template <int NT, int LOADER, int EPI>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(NT == 64 ? 4 : 2))) void k_pw_i16(PwArgs a) {
  using S = PwSmemIN<NT>;
  constexpr int RT = NT / 64;
  __shared__ __attribute__((aligned(1024))) char st0[S::STAGE];
  __shared__ __attribute__((aligned(1024))) char st1[S::STAGE];
  __shared__ __attribute__((aligned(1024))) char st2[S::STAGE];
  const int ntile = (a.P + 127) / 128;
  // (tile, row pass) pairs with the row pass fastest, each XCD taking a
  // contiguous range: the passes over one pixel tile run together and share
  // its activations in L2.
  const int npass = a.N / NT;
  const int lin = xcd_tile(blockIdx.x, gridDim.x);
  const int tile = lin / npass;
  if (tile >= ntile) return;
  const int lane = threadIdx.x & 63, h = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int pg = wave & 3, hf = wave >> 2;
  const int n0 = (lin - tile * npass) * NT;
  const int nk = a.K / 64;

  intx16 acc[RT][3];
#pragma unroll
  for (int t = 0; t < RT; ++t) acc[t][0] = acc[t][1] = acc[t][2] = intx16{};
  intx4 corr[RT][4];
#pragma unroll
  for (int t = 0; t < RT; ++t)
#pragma unroll
    for (int g = 0; g < 4; ++g) corr[t][g] = *(const intx4*)((const int*)a.bias + n0 + 32 * (hf * RT + t) + 8 * g + 4 * h);

  pwi_issue<NT, LOADER>(a, tile, n0, 0, st0, wave, lane);
  if (nk > 1) pwi_issue<NT, LOADER>(a, tile, n0, 1, st1, wave, lane);
  auto step = [&](int kc, const char* cur, char* refill) {
    const int ahead = min(nk - 1 - kc, 1);  // stages issued after kc still in flight
    if (ahead == 1) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(S::DMA_PER_WAVE) : "memory");
    else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    lds_barrier();
    if (kc + 2 < nk) pwi_issue<NT, LOADER>(a, tile, n0, kc + 2, refill, wave, lane);
    pwi_compute<NT, LOADER>(cur, pg, hf, lane, acc);
  };
  for (int kc = 0; kc < nk; kc += 3) {
    step(kc, st0, st2);
    if (kc + 1 < nk) step(kc + 1, st1, st0);
    if (kc + 2 < nk) step(kc + 2, st2, st1);
  }
  lds_barrier();

  // park the rescaled int16 results as int32, as in the fp16 kernel
  constexpr int SWZ = (NT / 4 - 1) & 31;
  // pixel group g parks at offset (g % GPS) * PARK of stage g / GPS
  constexpr int PARK = 32 * NT * 4, GPS = S::STAGE / PARK;
  static_assert(GPS >= 2, "four pixel groups fit three stage buffers");
  auto park = [&](int g) __attribute__((always_inline)) -> char* {
    return (g / GPS == 0 ? st0 : g / GPS == 1 ? st1 : st2) + (g % GPS) * PARK;
  };
  {
    char* ob = park(pg);
    const int row = lane & 31;
#pragma unroll
    for (int t = 0; t < RT; ++t)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int nl = 32 * (hf * RT + t) + 8 * g + 4 * h;
        intx4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = 4 * g + e;
          o[e] = rescale13(combine_i16(acc[t][0][r], acc[t][1][r], acc[t][2][r], corr[t][g][e]));
        }
        *(intx4*)(ob + row * (NT * 4) + (((nl >> 2) ^ (row & SWZ)) << 4)) = o;
      }
  }
  // prior head: a pass covers channels c0 .. c0+31 (rows 0-31 mu_i, 32-63 s_i);
  // the tile's symbols are staged in stage buffer 2 as [channel][pixel]
  const int c0 = n0 / 2;
  int16_t* qt = (int16_t*)st2;
  if constexpr (EPI == EP_PRIOR_DEC) {
    static_assert(NT == 64, "prior passes are 64 rows");
    const int ch = threadIdx.x >> 4, k = threadIdx.x & 15;
    const int p0 = tile * 128 + 8 * k;
    const int16_t* src = a.q_in + (size_t)(c0 + ch) * a.P + p0;
    shortx8 v = {};
    if ((a.P & 7) == 0 && p0 + 8 <= a.P) {
      v = *(const shortx8*)src;
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = p0 + e < a.P ? src[e] : (short)0;
    }
    *(shortx8*)(qt + ch * 128 + 8 * k) = v;
  }
  lds_barrier();

  auto parked = [&](int px, int nl8, int* v) {
    const int gpx = px >> 5, row = px & 31;
    const char* ob = park(gpx);
    const intx4 o0 = *(const intx4*)(ob + row * (NT * 4) + (((2 * nl8) ^ (row & SWZ)) << 4));
    const intx4 o1 = *(const intx4*)(ob + row * (NT * 4) + (((2 * nl8 + 1) ^ (row & SWZ)) << 4));
#pragma unroll
    for (int e = 0; e < 4; ++e) { v[e] = o0[e]; v[4 + e] = o1[e]; }
  };
  constexpr int UNITS = 128 * (NT / 8);
  if constexpr (EPI == EP_PRIOR || EPI == EP_PRIOR_DEC) {
    // thread = (pixel px, 8 channels g8): q = RHE((y_i - mu_i) / 512),
    // yhat_i = clip(512 q + mu_i), sigma from the table at s_i
    const int px = threadIdx.x >> 2, g8 = threadIdx.x & 3;
    const int gp = tile * 128 + px;
    const int c = c0 + 8 * g8;
    int mu[8], sv[8];
    parked(px, g8, mu);
    parked(px, 4 + g8, sv);
    if constexpr (EPI == EP_PRIOR) {
      double bsum = 0.0;
      shortx8 yv = {};
      if (gp < a.P) yv = *(const shortx8*)((const int16_t*)a.y + (size_t)gp * a.Cdst + c);
      shortx8 yh;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int q = rhe_shift((int)yv[e] - mu[e], 9);
        qt[(8 * g8 + e) * 128 + px] = (int16_t)q;
        yh[e] = (short)clip16(512 * q + mu[e]);
        if (gp < a.P) bsum += (double)symbol_bits((float)q, a.sigma_tab[sv[e] + 32768]);
      }
      if (gp < a.P) *(shortx8*)((int16_t*)a.dst + (size_t)gp * a.Cdst + c) = yh;
      __shared__ double red[8];
      bsum = wave_sum(bsum);
      if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = bsum;
      lds_barrier();
      {
        const int ch = threadIdx.x >> 4, k = threadIdx.x & 15;
        const int p0 = tile * 128 + 8 * k;
        const shortx8 v = *(const shortx8*)(qt + ch * 128 + 8 * k);
        int16_t* dq = a.q_out + (size_t)(c0 + ch) * a.P + p0;
        if ((a.P & 7) == 0 && p0 + 8 <= a.P) {
          *(shortx8*)dq = v;
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (p0 + e < a.P) dq[e] = v[e];
        }
      }
      if (threadIdx.x == 0) {
        double t = 0.0;
#pragma unroll
        for (int w = 0; w < 8; ++w) t += red[w];
        a.partials[(size_t)tile * npass + n0 / NT] = t;
      }
    } else {
      if (gp < a.P) {
        shortx8 yh;
#pragma unroll
        for (int e = 0; e < 8; ++e) yh[e] = (short)clip16(512 * (int)qt[(8 * g8 + e) * 128 + px] + mu[e]);
        *(shortx8*)((int16_t*)a.dst + (size_t)gp * a.Cdst + c) = yh;
      }
    }
  } else if constexpr (EPI == EP_REC) {
#pragma unroll
    for (int it = 0; it < UNITS / 512; ++it) {
      const int idx = it * 512 + threadIdx.x;
      const int nl8 = idx >> 7, px = idx & 127;
      const int gp = tile * 128 + px;
      if (gp < a.P) {
        int v[8];
        parked(px, nl8, v);
        const int n = n0 + 8 * nl8, c = n >> 6, i = (n >> 3) & 7;
        const int py = gp / a.w8, pxx = gp - py * a.w8;
        shortx8 o;
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] = (short)min(max(v[e], 0), 512);
        *(shortx8*)((int16_t*)a.dst + (size_t)c * a.H * a.W + (size_t)(8 * py + i) * a.W + 8 * pxx) = o;
      }
    }
  } else {
#pragma unroll
    for (int it = 0; it < UNITS / 512; ++it) {
      const int idx = it * 512 + threadIdx.x;
      const int px = idx / (NT / 8), nl8 = idx % (NT / 8);
      const int gp = tile * 128 + px;
      if (gp < a.P) {
        int v[8];
        parked(px, nl8, v);
        shortx8 o;
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] = (short)v[e];
        size_t off;
        if constexpr (EPI == EP_NHWC) {
          off = (size_t)gp * a.Cdst + n0 + 8 * nl8;
        } else {
          const int C = a.Cdst, n = n0 + 8 * nl8;
          const int sp = n / C, c = n - sp * C;
          const int w16 = a.w8 >> 1;
          const int Y = gp / w16, X = gp - Y * w16;
          off = (size_t)((2 * Y + (sp >> 1)) * a.w8 + 2 * X + (sp & 1)) * C + c;
        }
        *(shortx8*)((int16_t*)a.dst + off) = o;
      }
    }
  }
}

// Whole DC block on the integer path; same dataflow as the fp16 block kernel
// (8 waves per 8 x 16 pixel tile, LDS-staged halo and chunk-major weights,
// hidden chunks exchanged between the two waves of a pixel group), with every
// contraction done as int8 digit products:
//   pw1 (per hidden chunk): three accumulators hh, hl + lh, ll, combined and
//       rescaled once per chunk;
//   pw2 (per output tile and chunk): t = hh; t <<= 8; t += hl + lh (MFMA);
//       acc += t << 8; acc += ll (MFMA).  All in wrapping int32, which equals
//       the exact sum whenever that fits int32.
template <int C>
struct DcSmemI {
  static constexpr int KSI = C / 32, MT = C / 32, FR = 2 * KSI + 2 * MT, CHUNK = FR * 1024;
};

template <int C>
__device__ __forceinline__ void dci_issue(const char* wchunks, int j, char* buf, int wave, int lane) {
  constexpr int FR = DcSmemI<C>::FR;
#pragma unroll
  for (int i = 0; i < FR / 8; ++i) {
    const int f = wave + 8 * i;
    const char* g = wchunks + ((size_t)j * FR + f) * 1024 + lane * 16;
    dma16(g, buf + f * 1024);
  }
}

struct I16Acc {
  intx16 hh, mid, ll;
};

// pw1 for hidden chunk j; the low-digit accumulator starts at the chunk's
// correction 512 b_i + 128 sum w (row 8 g + 4 h + e of register 4 g + e).
template <int C>
__device__ __forceinline__ I16Acc dci_hidden_mfma(const char* wb, const intx4* ah, const intx4* al, const int* c1s,
                                                  int j, int h, int lane) {
  constexpr int KSI = DcSmemI<C>::KSI;
  const intx4* w = (const intx4*)wb + lane;
  // Fragment reads are issued ahead of the MFMAs in groups of half a chunk.
  constexpr int G = KSI >= 4 ? KSI / 2 : KSI;
  I16Acc acc{{}, {}, {}};
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const intx4 cv = *(const intx4*)(c1s + 32 * j + 8 * g + 4 * h);
#pragma unroll
    for (int e = 0; e < 4; ++e) acc.ll[4 * g + e] = cv[e];
  }
#pragma unroll
  for (int s0 = 0; s0 < KSI; s0 += G) {
    intx4 wa[G], wl[G];
#pragma unroll
    for (int s = 0; s < G; ++s) {
      wa[s] = w[(s0 + s) * 64];
      wl[s] = w[(KSI + s0 + s) * 64];
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int s = 0; s < G; ++s) {
      acc.hh = mfma_i8(wa[s], ah[s0 + s], acc.hh);
      acc.mid = mfma_i8(wa[s], al[s0 + s], acc.mid);
      acc.mid = mfma_i8(wl[s], ah[s0 + s], acc.mid);
      acc.ll = mfma_i8(wl[s], al[s0 + s], acc.ll);
    }
  }
  return acc;
}

// Combine, rescale, integer LeakyReLU (slope 819 / 8192), split into int8
// digits, store as the pw2 operand fragments.  The LeakyReLU is
// max(h, RHE(819 h / 2^13)): for h >= 0 the scaled value never exceeds h, for
// h < 0 it is never below h, so the maximum selects the right branch.
__device__ __forceinline__ void dci_hidden_store(const I16Acc& acc, int lane, intx4* gx) {
  int gv[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int hv = rescale13(combine_i16(acc.hh[r], acc.mid[r], acc.ll[r], 0));
    const int m = 819 * hv;  // |m| < 2^25: the bias form of RHE cannot overflow
    gv[r] = max(hv, (m + 4095 + ((m >> 13) & 1)) >> 13);
  }
  uint32_t d[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) d[e] = pack2(gv[2 * e], gv[2 * e + 1]);
  intx4 gh, gl;
  split16(d, gh, gl);
  gx[lane] = gh;
  gx[64 + lane] = gl;
}

template <int C>
__device__ __forceinline__ void dci_project(const char* wb, const intx4* gx, int hf, int lane, intx16* out) {
  constexpr int KSI = DcSmemI<C>::KSI, MT = DcSmemI<C>::MT;
  const intx4* w = (const intx4*)wb + lane;
  const intx4 gh = gx[lane], gl = gx[64 + lane];
#pragma unroll
  for (int t = 0; t < MT / 2; ++t) {
    const int tt = hf * (MT / 2) + t;
    const intx4 wa = w[(2 * KSI + tt) * 64], wl = w[(2 * KSI + MT + tt) * 64];
    intx16 v = mfma_i8(wa, gh, intx16{});
#pragma unroll
    for (int r = 0; r < 16; ++r) v[r] = (int)((uint32_t)v[r] << 8);
    v = mfma_i8(wa, gl, v);
    v = mfma_i8(wl, gh, v);
#pragma unroll
    for (int r = 0; r < 16; ++r) out[t][r] = (int)(((uint32_t)v[r] << 8) + (uint32_t)out[t][r]);
    out[t] = mfma_i8(wl, gl, out[t]);
  }
}

template <int C>
__global__ __launch_bounds__(512) void k_dcblock_i16(BlockArgs a) {
  constexpr int KSI = DcSmemI<C>::KSI;
  constexpr int NCH = 2 * C / 32;
  constexpr int MT = DcSmemI<C>::MT;
  constexpr int CHUNK = DcSmemI<C>::CHUNK;
  constexpr int LDS_PER_WAVE = DcSmemI<C>::FR / 8;
  constexpr int TH = 8, TW = 16;
  constexpr int HW = TW + 2;
  // Depthwise role: band sg of 4 tile rows x channel part cp (CP parts of CPC
  // channels); lane l = pixel (row 4 sg + l / 16, column l % 16).  With C = 64
  // there are only two parts and waves 4-7 sit the depthwise out.
  constexpr int CP = C / 32 < 4 ? C / 32 : 4;
  constexpr int CPC = C / CP;                  // channels per part
  constexpr int NG = CPC / 8;                  // 8-channel groups (16-byte vectors per halo pixel)
  constexpr int NS = CPC / 32;                 // 32-channel MFMA steps per part
  constexpr int BPX = 6 * HW;
  constexpr int RINSTR = (BPX * NG + 63) / 64;
  constexpr int REGION = 16 * 1024;
  constexpr int SWS = NG == 8 ? 0 : 1;         // vector v of pixel hp at v ^ ((hp >> SWS) & (NG-1))
  static_assert(NG == 4 || NG == 8, "C in {64, 128, 256}");
  static_assert(RINSTR * 1024 <= REGION && 4 * NS * 1024 <= REGION, "band and exchange fit a region");
  static_assert(NCH % 4 == 0, "chunk loop is unrolled by four");
  constexpr int BUF = CHUNK > 2 * REGION ? CHUNK : 2 * REGION;
  __shared__ __attribute__((aligned(1024))) char wb0[BUF];
  __shared__ __attribute__((aligned(1024))) char wb1[BUF];
  __shared__ __attribute__((aligned(1024))) char wb2[BUF];
  __shared__ __attribute__((aligned(1024))) char wb3[BUF];
  __shared__ intx4 gx0[4][128];
  __shared__ intx4 gx1[4][128];
  __shared__ __attribute__((aligned(16))) int c1s[2 * C];  // pw1 corrections 512 b + 128 sum w
  __shared__ __attribute__((aligned(16))) int c2s[C];      // pw2 corrections

  const int tiles_x = (a.w + TW - 1) / TW;
  const int ntile = tiles_x * ((a.h + TH - 1) / TH);
  const int tile = xcd_tile(blockIdx.x, gridDim.x);
  if (tile >= ntile) return;
  const int ty0 = (tile / tiles_x) * TH, tx0 = (tile % tiles_x) * TW;
  const int lane = threadIdx.x & 63, h = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int pg = wave & 3, hf = wave >> 2;
  const int sg = pg >> 1;
  const int cp = CP == 4 ? (wave & 1) | ((wave >> 2) << 1) : (wave & 1);
  const bool dw_on = CP == 4 || wave < 4;
  const int cb = cp * CPC;
  const int16_t* z = (const int16_t*)a.src;
  const char* wchunks = (const char*)a.w1;
  auto bufp = [&](int k) __attribute__((always_inline)) -> char* {
    return k == 0 ? wb0 : k == 1 ? wb1 : k == 2 ? wb2 : wb3;
  };
  auto region = [&](int sg_, int cp_) __attribute__((always_inline)) -> char* {
    return bufp(2 * (cp_ >> 1) + sg_) + (cp_ & 1) * REGION;
  };
  char* const own = region(sg, cp);

  // Corrections straight into LDS (waves 0 and 1, before their halo loads;
  // waited for with those loads and made visible by the exchange barrier).
  if (wave < 2) {
    const int* src = wave == 0 ? (const int*)a.b1 : (const int*)a.b2;
    int* dstl = wave == 0 ? c1s : c2s;
    const int n16 = (wave == 0 ? 2 * C : C) / 4;  // 16-byte units
#pragma unroll
    for (int i = 0; i < (2 * C / 4 + 63) / 64; ++i)
      if (64 * i + lane < n16) dma16(src + 4 * (64 * i + lane), dstl + 4 * 64 * i);
  }

  // Halo band (as in the fp16 block): slot S = 16-byte unit S of the region.
  if (dw_on) {
#pragma unroll
    for (int i = 0; i < RINSTR; ++i) {
      const int S = i * 64 + lane;
      const int hp = S / NG, v = (S % NG) ^ ((hp >> SWS) & (NG - 1));
      const int hy = ty0 - 1 + 4 * sg + hp / HW, hx = tx0 - 1 + hp % HW;
      const bool in = hp < BPX && hy >= 0 && hy < a.h && hx >= 0 && hx < a.w;
      dma16(in ? z + (size_t)(hy * a.w + hx) * C + cb + 8 * v : (const int16_t*)a.zpad, own + i * 1024);
    }
  }

  if (dw_on) {
    // Depthwise 3x3: exact int32 sums, one v_mad_i32_i16 per tap and channel
    // (op_sel picks the low or high int16 of the packed activation and of the
    // wave-uniform weight pair), bias 512 b_i, rescaled to int16.
    int tap_off[9];
#pragma unroll
    for (int ky = 0; ky < 3; ++ky)
#pragma unroll
      for (int kx = 0; kx < 3; ++kx) {
        const int hp = ((lane >> 4) + ky) * HW + (lane & 15) + kx;
        tap_off[ky * 3 + kx] = hp * (NG * 16) + (((hp >> SWS) & (NG - 1)) << 4);
      }
    cintx4* dww = (cintx4*)((const int16_t*)a.dww + cb);  // [9][C] int16, 8 per vector
    cint* dwb = (cint*)((const int*)a.dwb + cb);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this wave's band
    uint32_t dv[NG][4];
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      int acc[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] = dwb[8 * g + e];
#pragma unroll
      for (int t = 0; t < 9; ++t) {
        const intx4 zv = *(const intx4*)(own + (tap_off[t] ^ (g << 4)));
        const intx4 wv = dww[(t * C + 8 * g) / 8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int wp = wv[i];
          const int zi = zv[i];
          asm("v_mad_i32_i16 %0, %1, %2, %0" : "+v"(acc[2 * i]) : "v"(zi), "s"(wp));
          asm("v_mad_i32_i16 %0, %1, %2, %0 op_sel:[1,1,0,0]" : "+v"(acc[2 * i + 1]) : "v"(zi), "s"(wp));
        }
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) dv[g][i] = pack2(rescale13(acc[2 * i]), rescale13(acc[2 * i + 1]));
      __builtin_amdgcn_sched_barrier(0);  // one group's weights live at a time
    }
    // 16-channel unit u = groups 2u, 2u+1 -> hi / lo digit vectors; units 2p and
    // 2p+1 swap lane halves into the B fragments of step cb / 32 + p for pixel
    // groups 2 sg (lanes 0-31) and 2 sg + 1; they overwrite the dead band:
    // [pixel group & 1][step p][hi, lo] x 1 KiB.
#pragma unroll
    for (int p = 0; p < NS; ++p) {
      intx4 xh, xl, yh, yl;
      {
        uint32_t d[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) { d[i] = dv[4 * p][i]; d[4 + i] = dv[4 * p + 1][i]; }
        split16(d, xh, xl);
#pragma unroll
        for (int i = 0; i < 4; ++i) { d[i] = dv[4 * p + 2][i]; d[4 + i] = dv[4 * p + 3][i]; }
        split16(d, yh, yl);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const auto rh = __builtin_amdgcn_permlane32_swap((uint32_t)xh[i], (uint32_t)yh[i], false, false);
        xh[i] = (int)rh[0];
        yh[i] = (int)rh[1];
        const auto rl = __builtin_amdgcn_permlane32_swap((uint32_t)xl[i], (uint32_t)yl[i], false, false);
        xl[i] = (int)rl[0];
        yl[i] = (int)rl[1];
      }
      *(intx4*)(own + ((0 * NS + p) * 2 + 0) * 1024 + lane * 16) = xh;
      *(intx4*)(own + ((0 * NS + p) * 2 + 1) * 1024 + lane * 16) = xl;
      *(intx4*)(own + ((1 * NS + p) * 2 + 0) * 1024 + lane * 16) = yh;
      *(intx4*)(own + ((1 * NS + p) * 2 + 1) * 1024 + lane * 16) = yl;
    }
  }
  if (!dw_on) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // corrections (waves 0, 1 are depthwise waves)
  lds_barrier();

  // MFMA role: the digit fragments of all C filtered channels of this wave's 32 pixels
  intx4 ah[KSI], al[KSI];
#pragma unroll
  for (int s = 0; s < KSI; ++s) {
    const char* src = region(sg, s / NS) + (((pg & 1) * NS + s % NS) * 2) * 1024 + lane * 16;
    ah[s] = *(const intx4*)src;
    al[s] = *(const intx4*)(src + 1024);
  }
  lds_barrier();  // exchange read: the buffers take weight chunks from here on

  dci_issue<C>(wchunks, 0, wb0, wave, lane);
  dci_issue<C>(wchunks, 1, wb1, wave, lane);
  dci_issue<C>(wchunks, 2, wb2, wave, lane);

  intx16 out[MT / 2];
#pragma unroll
  for (int t = 0; t < MT / 2; ++t) out[t] = intx16{};

  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * LDS_PER_WAVE) : "memory");
  lds_barrier();  // chunk 0 staged; hidden chunk 0 runs while chunks 1 and 2 arrive
  if (hf == 0) dci_hidden_store(dci_hidden_mfma<C>(wb0, ah, al, c1s, 0, h, lane), lane, gx0[pg]);
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(LDS_PER_WAVE) : "memory");
  lds_barrier();  // chunk 1 staged, hidden chunk 0 visible

  // The residual tile (128 pixels x C int16, pixel px at byte 2 C px of
  // buffers 0 and 1) is loaded during the last two chunks.
  static_assert(128 * C * 2 <= 2 * BUF, "residual tile fits two buffers");
  auto issue_residual = [&]() __attribute__((always_inline)) {
    constexpr int CH8 = C / 8;
#pragma unroll
    for (int i = 0; i < C / 32; ++i) {
      const int k = wave + 8 * i;  // 1 KiB unit k of the tile
      const int S = k * 64 + lane;
      const int px = S / CH8, k8 = S % CH8;
      const int yy = ty0 + (px >> 4), xx = tx0 + (px & 15);
      const bool in = yy < a.h && xx < a.w;
      char* dstl = (k * 1024 < BUF ? wb0 : wb1) + (k * 1024) % BUF;
      dma16(in ? z + (size_t)(yy * a.w + xx) * C + 8 * k8 : (const int16_t*)a.zpad, dstl);
    }
  };
  auto step = [&](int j, const char* wcur, const char* wnxt, char* wiss, intx4* gcur, intx4* gnxt)
                  __attribute__((always_inline)) {
    const bool more = j + 3 < NCH;
    if (more) dci_issue<C>(wchunks, j + 3, wiss, wave, lane);
    const bool produce = j + 1 < NCH && hf == ((j + 1) & 1);
    I16Acc hacc;
    if (produce) hacc = dci_hidden_mfma<C>(wnxt, ah, al, c1s, j + 1, h, lane);
    if (j == NCH - 2) issue_residual();  // buffers 0 and 1 are free from here on
    dci_project<C>(wcur, gcur, hf, lane, out);
    if (produce) dci_hidden_store(hacc, lane, gnxt);
    if (more) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(LDS_PER_WAVE) : "memory");
    else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    lds_barrier();
  };
  for (int j = 0; j < NCH; j += 4) {
    step(j + 0, wb0, wb1, wb3, gx0[pg], gx1[pg]);
    step(j + 1, wb1, wb2, wb0, gx1[pg], gx0[pg]);
    step(j + 2, wb2, wb3, wb1, gx0[pg], gx1[pg]);
    step(j + 3, wb3, wb0, wb2, gx1[pg], gx0[pg]);
  }

  // Epilogue: rescale(sum + correction) to int16 in registers, parked in
  // buffers 2 (pixel groups 0, 1) and 3 (groups 2, 3), row = pixel, 8-byte unit
  // u of the row at u ^ (row & 15); then each thread adds the residual to 8
  // channels of one pixel with saturation and stores them with one 16-byte store.
  {
    char* ob = (pg < 2 ? wb2 : wb3) + (pg & 1) * (32 * C * 2);
    const int row = lane & 31;
#pragma unroll
    for (int t = 0; t < MT / 2; ++t)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int cc = 32 * (hf * (MT / 2) + t) + 8 * g + 4 * h;
        const intx4 cv = *(const intx4*)(c2s + cc);
        shortx4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = (short)rescale13((int)((uint32_t)out[t][4 * g + e] + (uint32_t)cv[e]));
        *(shortx4*)(ob + row * (C * 2) + (((cc >> 2) ^ (row & 15)) << 3)) = o;
      }
  }
  lds_barrier();  // the residual loads were waited for in the last chunk step
  constexpr int CH8 = C / 8;
  constexpr int PER = 128 * CH8 / 512;
  int16_t* dst = (int16_t*)a.dst;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int idx = i * 512 + threadIdx.x;
    const int px = idx / CH8, k8 = idx % CH8;
    const int row = px & 31;
    const int yy = ty0 + (px >> 4), xx = tx0 + (px & 15);
    if (yy < a.h && xx < a.w) {
      const char* ob = (px < 64 ? wb2 : wb3) + ((px >> 5) & 1) * (32 * C * 2) + row * (C * 2);
      const shortx4 p0 = *(const shortx4*)(ob + (((2 * k8) ^ (row & 15)) << 3));
      const shortx4 p1 = *(const shortx4*)(ob + (((2 * k8 + 1) ^ (row & 15)) << 3));
      const int rb = px * (C * 2) + 16 * k8;  // residual byte offset in buffers 0, 1
      const shortx8 zv = *(const shortx8*)((rb < BUF ? wb0 : wb1) + rb % BUF);
      shortx8 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        o[e] = (short)clip16((int)zv[e] + (int)p0[e]);
        o[4 + e] = (short)clip16((int)zv[4 + e] + (int)p1[e]);
      }
      // streaming store: the block's output is read by the next launch, not this one
      __builtin_nontemporal_store(o, (shortx8*)(dst + (size_t)(yy * a.w + xx) * C + 8 * k8));
    }
  }
}

template <int NT>
static hipError_t pw_dispatch(int loader, int epi, const PwArgs& a, hipStream_t st) {
  dim3 grid(grid_tiles(a.P) * (a.N / NT)), block(512);
#define NC_PW(L, E)                                                            \
  if (loader == L && epi == E) {                                               \
    launch(k_pw_i16<NT, L, E>, grid, block, st, a);                            \
    return hipGetLastError();                                                  \
  }
  NC_PW(LD_NHWC, EP_NHWC)
  NC_PW(LD_FRAME, EP_NHWC)
  NC_PW(LD_DOWN, EP_NHWC)
  NC_PW(LD_NHWC, EP_UP)
  NC_PW(LD_NHWC, EP_REC)
  NC_PW(LD_NHWC, EP_PRIOR)
  NC_PW(LD_NHWC, EP_PRIOR_DEC)
#undef NC_PW
  return hipErrorInvalidValue;
}

// 64 rows per workgroup pass: two workgroups fit a CU, and the passes over one
// pixel tile run side by side on one XCD.  K must be a multiple of 64 (C = 64,
// 128, 256; 192 for the patch embed) and N a multiple of 64.
hipError_t launch_pw_i16(int loader, int epi, const PwArgs& a, hipStream_t st) {
  if (a.K % 64 || a.N % 64) return hipErrorInvalidValue;
  return pw_dispatch<64>(loader, epi, a, st);
}

hipError_t launch_dcblock_i16(int C, const BlockArgs& a, hipStream_t st) {
  dim3 grid(dc_grid(a.h, a.w)), block(512);
  switch (C) {
    case 64: launch(k_dcblock_i16<64>, grid, block, st, a); break;
    case 128: launch(k_dcblock_i16<128>, grid, block, st, a); break;
    case 256: launch(k_dcblock_i16<256>, grid, block, st, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Integer prior head, quantiser q = RHE((y_i - mu_i) / 512),
// yhat_i = clip(512 q + mu_i) and bits with sigma looked up from the
// 65536-entry table indexed by s_i (Supp. B.2, Alg. 1), as the epilogue of the
// pointwise kernel over passes of 32 mu rows + the 32 s rows of the same
// channels.  Bit partial sums: one per (tile, pass).
int prior_partials_i16(int C, int P) { return ((P + 127) / 128) * (C / 32); }

hipError_t launch_prior_i16(const PriorArgs& pa, hipStream_t st, int* n_partials) {
  if (pa.C % 32) return hipErrorInvalidValue;
  PwArgs a;
  std::memset(&a, 0, sizeof(a));
  a.wfrag = pa.wfrag;
  a.wfrag_lo = pa.wfrag_lo;
  a.bias = pa.bias;
  a.K = pa.C;
  a.N = 2 * pa.C;
  a.P = pa.P;
  a.src0 = pa.yhat_prev;
  a.C0 = pa.C;
  a.dst = pa.yhat_new;
  a.Cdst = pa.C;
  a.y = pa.y;
  a.q_in = pa.q_in;
  a.q_out = pa.q_out;
  a.partials = pa.partials;
  a.sigma_tab = pa.sigma_tab;
  if (n_partials) *n_partials = prior_partials_i16(pa.C, pa.P);
  return pw_dispatch<64>(LD_NHWC, pa.decode ? EP_PRIOR_DEC : EP_PRIOR, a, st);
}

}  // namespace nc
