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

__device__ __forceinline__ uint32_t pack2(int lo, int hi) {
  return ((uint32_t)lo & 0xFFFFu) | ((uint32_t)hi << 16);
}

// The integer sigmoid table S (Sec. 4.5) from its compact form s8, and RHE of
// a / 512 (both described with the gated block below).
constexpr int kSigSat = 888;   // S[v] = 512 from here on
constexpr int kSigBytes = 896; // s8, padded to 16-byte units
__device__ __forceinline__ int dci_sigmoid(int v, const uint8_t* s8) {
  const int a = v < 0 ? -v : v;
  const int sa = a >= kSigSat ? 512 : 256 + (int)s8[min(a, kSigSat - 1)];  // index kept in the table
  return v < 0 ? 512 - sa : sa;
}
// RHE(m / 512) for |m| <= 2^30
__device__ __forceinline__ int rhe9(int m) { return (m + 255 + ((m >> 9) & 1)) >> 9; }

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
    if (k < a.C0) return (const char*)((const int16_t*)a.src0 + (size_t)gp * (a.ld0 ? a.ld0 : a.C0) + k);
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
    const int px = slot >> 3, v = (slot & 7) ^ ((px >> 1) & 7);  // conflict-free B reads (16-lane quarters)
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
      const half8 x0 = *(const half8*)(stage + pl * 128 + ((v0 ^ ((pl >> 1) & 7)) << 4));
      const half8 x1 = *(const half8*)(stage + pl * 128 + (((v0 + 1) ^ ((pl >> 1) & 7)) << 4));
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        d[e] = pack2(clip16((int)rintf((float)x0[2 * e] * 512.f)), clip16((int)rintf((float)x0[2 * e + 1] * 512.f)));
        d[4 + e] = pack2(clip16((int)rintf((float)x1[2 * e] * 512.f)), clip16((int)rintf((float)x1[2 * e + 1] * 512.f)));
      }
    } else {
      const intx4 q0 = *(const intx4*)(stage + pl * 128 + ((v0 ^ ((pl >> 1) & 7)) << 4));
      const intx4 q1 = *(const intx4*)(stage + pl * 128 + (((v0 + 1) ^ ((pl >> 1) & 7)) << 4));
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
  // the upsample that follows the prior in an encode: workgroup 0 first adds
  // up the frame's rate partials
  if constexpr (EPI == EP_UP)
    if (a.bits_out && blockIdx.x == 0) block_sum_to(a.sum_base, a.n_sum, a.bits_out);
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
  const int c0 = a.c_off + n0 / 2;
  int16_t* qt = (int16_t*)st2;
  uint8_t* kt = (uint8_t*)(st2 + 8192);  // scale indices, [channel][pixel]
  // planar store of the staged scale indices (after a barrier)
  auto store_k = [&]() __attribute__((always_inline)) {
    const int ch = threadIdx.x >> 4, k = threadIdx.x & 15;
    const int p0 = tile * 128 + 8 * k;
    uint8_t* dk = a.k_out + (size_t)(c0 + ch) * a.P + p0;
    const uint8_t* sk = kt + ch * 128 + 8 * k;
    if ((a.P & 7) == 0 && p0 + 8 <= a.P && ((uintptr_t)a.k_out & 7) == 0) {
      *(uint64_t*)dk = *(const uint64_t*)sk;
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (p0 + e < a.P) dk[e] = sk[e];
    }
  };
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
  // (mu_i, s_i) of 8 channels c .. c + 7 of pixel gp: the head's rows plus,
  // saturating, the addend of the two-step entropy model (hyper parameters,
  // or the first step's (mu_i, s_i) for the second step)
  auto prior_ms = [&](int px, int g8, int gp, int* mu, int* sv) __attribute__((always_inline)) {
    parked(px, g8, mu);
    parked(px, 4 + g8, sv);
    if (a.add && gp < a.P) {
      const size_t at = (size_t)gp * a.add_ld + (c0 + 8 * g8 - a.add_c0);
      const shortx8 hm = *(const shortx8*)((const int16_t*)a.add + at);
      const shortx8 hs = *(const shortx8*)((const int16_t*)a.add + at + a.add_s);
#pragma unroll
      for (int e = 0; e < 8; ++e) { mu[e] = clip16(mu[e] + (int)hm[e]); sv[e] = clip16(sv[e] + (int)hs[e]); }
    }
  };
  // channels >= split: (mu_i, s_i) go to the base buffer for the second step
  const bool to_base = a.split && c0 >= a.split;
  auto store_base = [&](int g8, int gp, const int* mu, const int* sv) __attribute__((always_inline)) {
    if (gp >= a.P) return;
    const int nb = a.Cdst - a.split;
    int16_t* b = (int16_t*)a.base + (size_t)gp * 2 * nb + (c0 + 8 * g8 - a.split);
    shortx8 m, v;
#pragma unroll
    for (int e = 0; e < 8; ++e) { m[e] = (short)mu[e]; v[e] = (short)sv[e]; }
    *(shortx8*)b = m;
    *(shortx8*)(b + nb) = v;
  };
  if constexpr (EPI == EP_SCALES) {
    const int px = threadIdx.x >> 2, g8 = threadIdx.x & 3;
    const int gp = tile * 128 + px;
    int mu[8], sv[8];
    prior_ms(px, g8, gp, mu, sv);
    if (to_base) {
      store_base(g8, gp, mu, sv);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) kt[(8 * g8 + e) * 128 + px] = a.k_tab[sv[e] + 32768];
      // mu_i (int16, NHWC), for yhat_i = clip(512 q + mu_i) once the symbols are decoded
      if (a.dst && gp < a.P) {
        shortx8 m;
#pragma unroll
        for (int e = 0; e < 8; ++e) m[e] = (short)mu[e];
        *(shortx8*)((int16_t*)a.dst + (size_t)gp * a.Cdst + c0 + 8 * g8) = m;
      }
    }
    lds_barrier();
    if (!to_base) store_k();
  } else if constexpr (EPI == EP_PRIOR || EPI == EP_PRIOR_DEC) {
    // thread = (pixel px, 8 channels g8): q = RHE((y_i - mu_i) / 512),
    // yhat_i = clip(512 q + mu_i), sigma from the table at s_i
    const int px = threadIdx.x >> 2, g8 = threadIdx.x & 3;
    const int gp = tile * 128 + px;
    const int c = c0 + 8 * g8;
    int mu[8], sv[8];
    prior_ms(px, g8, gp, mu, sv);
    if (to_base) {
      store_base(g8, gp, mu, sv);
      if constexpr (EPI == EP_PRIOR)
        if (threadIdx.x == 0) a.partials[(size_t)tile * npass + n0 / NT] = 0.0;
    } else if constexpr (EPI == EP_PRIOR) {
      double bsum = 0.0;
      shortx8 yv = {};
      if (gp < a.P) yv = *(const shortx8*)((const int16_t*)a.y + (size_t)gp * a.Cdst + c);
      shortx8 yh;
      if (a.k_out) {
#pragma unroll
        for (int e = 0; e < 8; ++e) kt[(8 * g8 + e) * 128 + px] = a.k_tab[sv[e] + 32768];
      }
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
      if (a.k_out) store_k();
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
  } else if constexpr (EPI == EP_ZQUANT) {
    // the 64 rows are the channels of z_i: q_z = RHE(z_i / 512) (staged
    // [channel][pixel] in stage buffer 2, 16 KiB), zhat_i = clip(512 q_z)
    // (NHWC), rate under sigma_z[c]
    static_assert(NT == 64, "z has 64 channels");
    const int px = threadIdx.x >> 2, g8 = threadIdx.x & 3;
    const int gp = tile * 128 + px;
    double bsum = 0.0;
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      const int cz = 32 * half + 8 * g8;
      int zv[8];
      parked(px, 4 * half + g8, zv);
      shortx8 zh;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int q = rhe_shift(zv[e], 9);
        qt[(cz + e) * 128 + px] = (int16_t)q;
        zh[e] = (short)clip16(512 * q);
        if (gp < a.P) bsum += (double)symbol_bits((float)q, a.zsigma[cz + e]);
      }
      if (gp < a.P) *(shortx8*)((int16_t*)a.dst + (size_t)gp * a.Cdst + cz) = zh;
    }
    __shared__ double redz[8];
    bsum = wave_sum(bsum);
    if ((threadIdx.x & 63) == 0) redz[threadIdx.x >> 6] = bsum;
    lds_barrier();
#pragma unroll
    for (int it = 0; it < 2; ++it) {
      const int ch = 32 * it + (threadIdx.x >> 4), k = threadIdx.x & 15;
      const int p0 = tile * 128 + 8 * k;
      const shortx8 v = *(const shortx8*)(qt + ch * 128 + 8 * k);
      int16_t* dq = a.q_out + (size_t)ch * a.P + p0;
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
      for (int w = 0; w < 8; ++w) t += redz[w];
      a.partials[tile] = t;
    }
  } else if constexpr (EPI == EP_GATE) {
    // rows 64 j .. + 31 of the pass: h1 of gated channels n0 / 2 + 32 j .. + 31,
    // rows 64 j + 32 .. + 63: the matching h2.  As the fused gated block:
    // WSiLU_i = RHE(h1 S[h1] / 512), g = clip(RHE(WSiLU_i h2 / 512)).
    constexpr int G = NT / 64, GU = 128 * G * 4;  // units (pixel, group, 8 channels)
#pragma unroll
    for (int it = 0; it < GU / 512; ++it) {
      const int idx = it * 512 + threadIdx.x;
      const int px = idx / (4 * G), j = (idx >> 2) % G, g8 = idx & 3;
      const int gp = tile * 128 + px;
      if (gp < a.P) {
        int h1[8], h2[8];
        parked(px, 8 * j + g8, h1);
        parked(px, 8 * j + 4 + g8, h2);
        shortx8 o;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int w1 = rhe9(h1[e] * dci_sigmoid(h1[e], a.sig8));  // |h S| <= 2^24
          o[e] = (short)clip16(rhe9(w1 * h2[e]));                    // |product| <= 2^30
        }
        *(shortx8*)((int16_t*)a.dst + (size_t)gp * a.Cdst + n0 / 2 + 32 * j + 8 * g8) = o;
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
        if constexpr (EPI == EP_LRELU) {
          // integer LeakyReLU, slope RHE(0.1 * 2^13) = 819: max(h, RHE(819 h / 2^13))
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int m = 819 * v[e];
            o[e] = (short)max(v[e], (m + 4095 + ((m >> 13) & 1)) >> 13);
          }
        } else if constexpr (EPI == EP_RESID) {
          // saturating residual add
          const shortx8 zr = *(const shortx8*)((const int16_t*)a.res + (size_t)gp * a.Cdst + n0 + 8 * nl8);
#pragma unroll
          for (int e = 0; e < 8; ++e) o[e] = (short)clip16((int)zr[e] + v[e]);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) o[e] = (short)v[e];
        }
        size_t off;
        if constexpr (EPI == EP_NHWC || EPI == EP_LRELU || EPI == EP_RESID) {
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

// Gated form (Supp. B.1, WSiLU and Chunk; Sec. 4.5, the sigmoid table).  With
// h = rescale(pw1 sum) on the int16 scale, WSiLU(h1) = RHE(h1 S[h1] / 512) and
// g = clip(RHE(WSiLU(h1) h2 / 512)), S[v] = RHE(512 sigmoid(4 v / 512)).  S is
// read from the compact LDS table s8: S[v] = 256 + s8[v] for 0 <= v < 888,
// 512 for v >= 888, and 512 - S[-v] for v < 0 (the table is odd about 256).
// WSiLU of the rescaled h1 chain, as 8 packed int16 pairs.
__device__ __forceinline__ void dci_wsilu(const I16Acc& acc, const uint8_t* s8, uint32_t* ws) {
  int wv[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int hv = rescale13(combine_i16(acc.hh[r], acc.mid[r], acc.ll[r], 0));
    wv[r] = rhe9(hv * dci_sigmoid(hv, s8));  // |h S| <= 2^24, |WSiLU| <= |h|
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) ws[e] = pack2(wv[2 * e], wv[2 * e + 1]);
}

// g = clip(RHE(WSiLU(h1) h2 / 512)) from the h2 chain, split into int8 digits
// and stored as the pw2 operand fragments (as dci_hidden_store).
__device__ __forceinline__ void dci_gate_store(const uint32_t* ws, const I16Acc& acc, int lane, intx4* gx) {
  int gv[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int h2 = rescale13(combine_i16(acc.hh[r], acc.mid[r], acc.ll[r], 0));
    const int w1 = (int)(short)(ws[r >> 1] >> (16 * (r & 1)));
    gv[r] = clip16(rhe9(w1 * h2));  // |product| <= 2^30
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

// Depthwise geometry of the integer DC block for C channels: wave w filters
// NCW channels (block w % NCB) over NRW tile rows (block w / NCB); lane =
// channel quad cq (fastest) x column slice colq of CPL columns, with its 9
// tap weights (int16 pairs) in registers and a sliding 3 x 3 window.  The
// wave's halo band ((NRW + 2) x 18 pixels x NCW channels) sits in its own LDS
// region, halo pixel hp at position hp ^ ((hp >> SWZ) & 1) so that the column
// slices of one 16-lane read group hit different banks when a pixel's slice is
// shorter than 128 bytes.  With C = 256 a wave takes 64 channels (whole
// 128-byte lines per halo pixel for its direct loads).
template <int C>
struct DcDwI {
  static constexpr int NCW = C == 256 ? 64 : 32;      // channels per wave
  static constexpr int NRW = C / NCW;                 // tile rows per wave
  static constexpr int NCB = C / NCW;                 // channel blocks
  static constexpr int NCQ = NCW / 4;                 // channel quads
  static constexpr int NCOLQ = 64 / NCQ;              // column slices
  static constexpr int CPL = 16 / NCOLQ;              // columns per lane
  static constexpr int SWZ = CPL == 4 ? 2 : 1;
  static constexpr int BP = (NRW + 2) * 18;           // halo pixels of the band
  static constexpr int UPP = NCW / 8;                 // 16-byte units per halo pixel
  static constexpr int SLOTS = BP * UPP;
  static constexpr int RINSTR = (SLOTS + 63) / 64;    // direct loads per wave for the band
  static constexpr int RB = SLOTS * 16;               // region bytes
  static constexpr int XF = 1024 + 16;                // exchange fragment stride (padded against bank conflicts)
  static constexpr int SPW = NCW / 32;                // 32-channel MFMA steps per wave
  static_assert(NCB * (8 / NRW) == 8 && NCOLQ * CPL == 16 && NRW % 2 == 0, "C in {64, 128, 256}");
  static_assert(2 * SPW * (NRW / 2) * XF <= RB, "the exchange fits the band's region");
};

// GATED: the gated form, scheduled like the fp16 kernel's: the weight entries
// alternate between the h1 rows and the h2 rows (plus the pw2 fragments) of
// one 32-channel pair, one wave of each SIMD pair produces both chains of a
// pair, keeps WSiLU(h1) in registers and gates when h2 is done; pw2 runs in odd
// iterations only.  The compact sigmoid table sits after the corrections.
template <int C, bool GATED>
__global__ __launch_bounds__(512) void k_dcblock_i16(BlockArgs a) {
  using G = DcDwI<C>;
  constexpr int KSI = DcSmemI<C>::KSI;
  constexpr int NCH = 2 * C / 32;
  constexpr int MT = DcSmemI<C>::MT;
  constexpr int FR = DcSmemI<C>::FR;
  constexpr int LDS_PER_WAVE = FR / 8;
  constexpr int TH = 8, TW = 16;
  static_assert(NCH % 4 == 0 && FR % 8 == 0, "chunk loop is unrolled by four");
  // LDS: chunk buffers 0-3, the hidden-chunk buffers, the corrections.  The
  // eight band regions start after the pw1 part (fragments 0 .. 2 KSI - 1) of
  // buffer 1 and are laid over the rest, which is dead once the filtered
  // channels have been exchanged: chunk 0 and the pw1 part of chunk 1 are
  // loaded from the start, the pw2 part of chunk 1 after the exchange.  After
  // the loop buffers 0-1 hold the residual tile and buffers 2-3 the parked
  // output.
  constexpr int BUF = DcSmemI<C>::CHUNK;
  constexpr int O1 = BUF, O2 = 2 * BUF, O3 = 3 * BUF, OGX = 4 * BUF;
  constexpr int OR = BUF + 2 * KSI * 1024;  // first band region
  constexpr int OC = (OR + 8 * G::RB > OGX + 16384 ? OR + 8 * G::RB : OGX + 16384);
  constexpr int SMEM = OC + 3 * C * 4 + (GATED ? kSigBytes : 0);  // c1s: 2 C ints, c2s: C ints, s8
  static_assert(SMEM <= 160 * 1024, "fits the LDS of a CU");
  __shared__ __attribute__((aligned(1024))) char smem[SMEM];
  char* const wb0 = smem;
  char* const wb1 = smem + O1;
  char* const wb2 = smem + O2;
  char* const wb3 = smem + O3;
  intx4* const gx0 = (intx4*)(smem + OGX);         // [pixel group][2 fragments x 64 lanes], even chunks
  intx4* const gx1 = (intx4*)(smem + OGX + 8192);  // odd chunks
  int* const c1s = (int*)(smem + OC);              // pw1 corrections 512 b + 128 sum w
  int* const c2s = c1s + 2 * C;                    // pw2 corrections
  const uint8_t* const s8 = (const uint8_t*)(c2s + C);  // gated: compact sigmoid table

  const int tiles_x = (a.w + TW - 1) / TW;
  const int ntile = tiles_x * ((a.h + TH - 1) / TH);
  const int tile = xcd_tile(blockIdx.x, gridDim.x);
  if (tile >= ntile) return;
  const int ty0 = (tile / tiles_x) * TH, tx0 = (tile % tiles_x) * TW;
  const int lane = threadIdx.x & 63, h = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int pg = wave & 3, hf = wave >> 2;
  const int16_t* z = (const int16_t*)a.src;
  const char* wchunks = (const char*)a.w1;
  auto region = [&](int w_) __attribute__((always_inline)) -> char* { return smem + OR + w_ * G::RB; };

  // Corrections straight into LDS (waves 0 and 1, before their bands: waited
  // for with them and made visible by the exchange barrier).
  if (wave < 2) {
    const int* src = wave == 0 ? (const int*)a.b1 : (const int*)a.b2;
    int* dstl = wave == 0 ? c1s : c2s;
    const int n16 = (wave == 0 ? 2 * C : C) / 4;  // 16-byte units
#pragma unroll
    for (int i = 0; i < (2 * C / 4 + 63) / 64; ++i)
      if (64 * i + lane < n16) dma16(src + 4 * (64 * i + lane), dstl + 4 * 64 * i);
  }
  if constexpr (GATED)  // wave 2, likewise
    if (wave == 2 && lane < kSigBytes / 16) dma16((const char*)a.sig8 + 16 * lane, (char*)(c2s + C));

  // Depthwise role.
  const int cbk = wave % G::NCB, rbk = wave / G::NCB;
  const int cq = lane % G::NCQ, colq = lane / G::NCQ;
  char* const own = region(wave);
  // this quad's 9 taps (int16 pairs) and four 512 b biases: 96 bytes per quad,
  // 22 words loaded (a loaded word left unused would be reused as a temporary
  // by the compiler, which then waits for this load before the band is issued)
  uint32_t wq[18];
  int bq[4];
  {
    const intx4* wsrc = (const intx4*)a.dww + 6 * (cbk * G::NCQ + cq);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const intx4 v = wsrc[i];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int x = v[e];
        wq[4 * i + e] = (uint32_t)x;
      }
    }
    const intx4 v4 = wsrc[4];
    const intx2 v5 = *(const intx2*)(wsrc + 5);
    const int x0 = v4[0], x1 = v4[1], x2 = v4[2], x3 = v4[3], x4 = v5[0], x5 = v5[1];
    wq[16] = (uint32_t)x0;
    wq[17] = (uint32_t)x1;
    bq[0] = x2;
    bq[1] = x3;
    bq[2] = x4;
    bq[3] = x5;
  }
  // Halo band: slot S = 16-byte unit S of the region holds unit S % UPP of
  // halo pixel pos(S / UPP); out-of-image pixels read the zero row.
  auto pos = [&](int hp) __attribute__((always_inline)) { return hp ^ ((hp >> G::SWZ) & 1); };
#pragma unroll
  for (int i = 0; i < G::RINSTR; ++i) {
    const int S = i * 64 + lane;
    if (G::SLOTS % 64 == 0 || S < G::SLOTS) {
      const int hp = pos(S / G::UPP), u = S % G::UPP;
      const int hy = ty0 + rbk * G::NRW - 1 + hp / 18, hx = tx0 - 1 + hp % 18;
      const bool in = hy >= 0 && hy < a.h && hx >= 0 && hx < a.w;
      dma16(in ? z + (size_t)(hy * a.w + hx) * C + cbk * G::NCW + 8 * u : (const int16_t*)a.zpad, own + i * 1024);
    }
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this wave's band (and the corrections)

  // Chunk 0 and the pw1 part of chunk 1 (consumed after the depthwise) are
  // requested a few fragments per output row, behind the band.  Load m < NP0
  // is fragment wave + 8 m of chunk 0, the others fragment wave + 8 (m - NP0)
  // of chunk 1.
  constexpr int NP0 = FR / 8, NP1 = (2 * KSI + 7) / 8;
  constexpr int PER_ROW = (NP0 + NP1 + G::NRW - 1) / G::NRW;
  auto issue_early = [&](int n) __attribute__((always_inline)) {
#pragma unroll
    for (int m = n * PER_ROW; m < (n + 1) * PER_ROW && m < NP0 + NP1; ++m) {
      const int c1 = m >= NP0;
      const int f = wave + 8 * (c1 ? m - NP0 : m);
      if (f < (c1 ? 2 * KSI : FR))
        dma16(wchunks + ((size_t)c1 * FR + f) * 1024 + lane * 16, (c1 ? wb1 : wb0) + f * 1024);
    }
  };

  // Depthwise 3x3: every band value this lane needs first (4 channels per
  // read), then the sliding window with exact int32 sums, one v_mad_i32_i16
  // per tap and channel (op_sel picks the low or high int16 of the packed
  // activation and weight), bias 512 b, rescaled to int16.
  uint32_t v[G::NRW + 2][G::CPL + 2][2];
#pragma unroll
  for (int y = 0; y < G::NRW + 2; ++y)
#pragma unroll
    for (int x = 0; x < G::CPL + 2; ++x) {
      const intx2 r = *(const intx2*)(own + pos(y * 18 + colq * G::CPL + x) * (G::UPP * 16) + cq * 8);
      const int r0 = r[0], r1 = r[1];
      v[y][x][0] = (uint32_t)r0;
      v[y][x][1] = (uint32_t)r1;
    }
  // The filtered quad is split into int8 digits and written straight into the
  // MFMA B fragments of its pixel group and 32-channel step, in this wave's
  // region (the band is dead once read): fragment (row pair j, step i, digit
  // d) at ((j SPW + i) 2 + d) XF; lane (pixel & 31) + 32 (bit 4 of the
  // channel), word (channel & 15) / 4.
  const int xhalf = (cq >> 2) & 1;
#pragma unroll
  for (int rr = 0; rr < G::NRW; ++rr)
#pragma unroll
    for (int k = 0; k < G::CPL; ++k) {
      int acc[4] = {bq[0], bq[1], bq[2], bq[3]};
#pragma unroll
      for (int ky = 0; ky < 3; ++ky)
#pragma unroll
        for (int kx = 0; kx < 3; ++kx) {
          const int t = 3 * ky + kx;
#pragma unroll
          for (int e = 0; e < 2; ++e) {
            const uint32_t zz = v[rr + ky][k + kx][e], ww = wq[2 * t + e];
            asm("v_mad_i32_i16 %0, %1, %2, %0" : "+v"(acc[2 * e]) : "v"(zz), "v"(ww));
            asm("v_mad_i32_i16 %0, %1, %2, %0 op_sel:[1,1,0,0]" : "+v"(acc[2 * e + 1]) : "v"(zz), "v"(ww));
          }
        }
      uint32_t dh, dl;
      split4(pack2(rescale13(acc[0]), rescale13(acc[1])), pack2(rescale13(acc[2]), rescale13(acc[3])), dh, dl);
      const int px = 16 * (rr & 1) + colq * G::CPL + k;  // pixel within the 32-pixel group
      const int f = ((rr >> 1) * G::SPW + (cq >> 3)) * 2;
      char* o = own + (px + 32 * xhalf) * 16 + (cq & 3) * 4;
      *(uint32_t*)(o + f * G::XF) = dh;
      *(uint32_t*)(o + (f + 1) * G::XF) = dl;
      if (k == G::CPL - 1) issue_early(rr);
    }
  lds_barrier();

  // MFMA role: the digit fragments of all C filtered channels of this wave's 32 pixels
  intx4 ah[KSI], al[KSI];
#pragma unroll
  for (int s = 0; s < KSI; ++s) {
    const int wcb = s / G::SPW, wrb = (2 * pg) / G::NRW;  // writer wave's channel and row blocks
    const int f = ((pg - wrb * (G::NRW / 2)) * G::SPW + (s - wcb * G::SPW)) * 2;
    const char* src = region(wrb * G::NCB + wcb) + lane * 16;
    ah[s] = *(const intx4*)(src + f * G::XF);
    al[s] = *(const intx4*)(src + (f + 1) * G::XF);
  }
  lds_barrier();  // exchange read: the regions take buffers 2, 3 and the hidden chunks from here on

  // the pw2 part of chunk 1 (2 MT fragments), then chunk 2
#pragma unroll
  for (int i = 0; i < (2 * MT + 7) / 8; ++i) {
    const int f = 2 * KSI + wave + 8 * i;
    if ((2 * MT) % 8 == 0 || f < FR) dma16(wchunks + ((size_t)FR + f) * 1024 + lane * 16, wb1 + f * 1024);
  }
  dci_issue<C>(wchunks, 2, wb2, wave, lane);

  // pw2 accumulators start at the correction 512 b + 128 sum w (wrapping int32
  // addition is associative, so the sum is the same as adding it at the end)
  intx16 out[MT / 2];
#pragma unroll
  for (int t = 0; t < MT / 2; ++t)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const intx4 cv = *(const intx4*)(c2s + 32 * (hf * (MT / 2) + t) + 8 * g + 4 * h);
#pragma unroll
      for (int e = 0; e < 4; ++e) out[t][4 * g + e] = cv[e];
    }

  // chunk 0 and the pw1 part of chunk 1 (the rest of chunk 1 and chunk 2 in flight)
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * MT / 8 + LDS_PER_WAVE) : "memory");
  lds_barrier();
  uint32_t ws[8];  // gated: WSiLU of the h1 chain of the pair being produced
  if (hf == 0) {
    if constexpr (GATED) dci_wsilu(dci_hidden_mfma<C>(wb0, ah, al, c1s, 0, h, lane), s8, ws);
    else dci_hidden_store(dci_hidden_mfma<C>(wb0, ah, al, c1s, 0, h, lane), lane, gx0 + 128 * pg);
  }
  lds_barrier();  // hidden chunk 0 visible

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
    // producer of chunk c: wave c % 2 of the pair, or in the gated form (c / 2) % 2
    const bool produce = j + 1 < NCH && hf == (GATED ? ((j + 1) >> 1) & 1 : (j + 1) & 1);
    I16Acc hacc;
    if (produce) {
      __builtin_amdgcn_s_setprio(2);  // the producer's chain first on the SIMD
      hacc = dci_hidden_mfma<C>(wnxt, ah, al, c1s, j + 1, h, lane);
    }
    if (j == NCH - 2) issue_residual();  // buffers 0 and 1 are free from here on
    if (!GATED || (j & 1)) dci_project<C>(wcur, gcur, hf, lane, out);
    if (produce) {
      if constexpr (GATED) {
        if ((j + 1) & 1) dci_gate_store(ws, hacc, lane, gnxt);  // h2 of the pair: gate it
        else dci_wsilu(hacc, s8, ws);
      } else {
        dci_hidden_store(hacc, lane, gnxt);
      }
    }
    if (more) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(LDS_PER_WAVE) : "memory");
    else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_setprio(0);
    lds_barrier();
  };
  for (int j = 0; j < NCH; j += 4) {
    step(j + 0, wb0, wb1, wb3, gx0 + 128 * pg, gx1 + 128 * pg);
    step(j + 1, wb1, wb2, wb0, gx1 + 128 * pg, gx0 + 128 * pg);
    step(j + 2, wb2, wb3, wb1, gx0 + 128 * pg, gx1 + 128 * pg);
    step(j + 3, wb3, wb0, wb2, gx1 + 128 * pg, gx0 + 128 * pg);
  }

  // Epilogue: rescale(sum) to int16 in registers (the sums started at the
  // corrections), parked in
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
        shortx4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = (short)rescale13(out[t][4 * g + e]);
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
  NC_PW(LD_NHWC, EP_LRELU)
  NC_PW(LD_NHWC, EP_RESID)
  NC_PW(LD_NHWC, EP_GATE)
  if constexpr (NT == 64) {  // epilogues that pair two 32-row halves of a pass
    NC_PW(LD_NHWC, EP_PRIOR)
    NC_PW(LD_NHWC, EP_PRIOR_DEC)
    NC_PW(LD_NHWC, EP_SCALES)
    NC_PW(LD_DOWN, EP_ZQUANT)
  }
#undef NC_PW
  return hipErrorInvalidValue;
}

// 64 rows per workgroup pass: two workgroups fit a CU, and the passes over one
// pixel tile run side by side on one XCD.  K must be a multiple of 64 (C = 64,
// 128, 256; 192 for the patch embed) and N a multiple of 64.
hipError_t launch_pw_i16(int loader, int epi, const PwArgs& a, hipStream_t st) {
  if (a.K % 64 || a.N % 64) return hipErrorInvalidValue;
  // 128 rows per pass for the patch embed and the 2C -> C fuse: their activation
  // tiles are the widest (K = 192 frame values or 2C channels), so halving the
  // passes that re-stage them pays, and they still have two passes per tile.
  if (a.N % 128 == 0 && epi == EP_NHWC && (loader == LD_FRAME || (loader == LD_NHWC && a.K >= 512)))
    return pw_dispatch<128>(loader, epi, a, st);
  // the two halves of a wide DC block (C > 256) at 1/8 scale: 128-row passes
  if ((epi == EP_LRELU || epi == EP_RESID || epi == EP_GATE) && a.N % 128 == 0)
    return pw_dispatch<128>(loader, epi, a, st);
  return pw_dispatch<64>(loader, epi, a, st);
}

hipError_t launch_dcblock_i16(int C, bool gated, const BlockArgs& a, hipStream_t st) {
  dim3 grid(dc_grid(a.h, a.w)), block(512);
  if (gated && !a.sig8) return hipErrorInvalidValue;
  switch (C * 2 + (gated ? 1 : 0)) {
    case 128: launch(k_dcblock_i16<64, false>, grid, block, st, a); break;
    case 256: launch(k_dcblock_i16<128, false>, grid, block, st, a); break;
    case 512: launch(k_dcblock_i16<256, false>, grid, block, st, a); break;
    case 129: launch(k_dcblock_i16<64, true>, grid, block, st, a); break;
    case 257: launch(k_dcblock_i16<128, true>, grid, block, st, a); break;
    case 513: launch(k_dcblock_i16<256, true>, grid, block, st, a); break;
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
  a.K = pa.K ? pa.K : pa.C;
  a.N = pa.N ? pa.N : 2 * pa.C;
  a.ld0 = pa.ld0;
  a.c_off = pa.c_off;
  a.add = pa.add;
  a.add_ld = pa.add_ld;
  a.add_s = pa.add_s;
  a.add_c0 = pa.add_c0;
  a.split = pa.split;
  a.base = pa.base;
  a.P = pa.P;
  a.src0 = pa.yhat_prev;
  a.C0 = a.K;
  a.dst = pa.decode == 2 ? pa.mu_out : pa.yhat_new;
  a.Cdst = pa.C;
  a.y = pa.y;
  a.q_in = pa.q_in;
  a.q_out = pa.q_out;
  a.partials = pa.partials;
  a.sigma_tab = pa.sigma_tab;
  a.k_out = pa.k_out;
  a.k_tab = pa.k_tab;
  if (n_partials) *n_partials = ((pa.P + 127) / 128) * (a.N / 64);
  return pw_dispatch<64>(LD_NHWC, pa.decode == 2 ? EP_SCALES : pa.decode ? EP_PRIOR_DEC : EP_PRIOR, a, st);
}

hipError_t launch_zquant_i16(const PwArgs& a, hipStream_t st, int* n_partials) {
  if (a.N != 64 || a.K % 64) return hipErrorInvalidValue;
  if (n_partials) *n_partials = (a.P + 127) / 128;
  return pw_dispatch<64>(LD_DOWN, EP_ZQUANT, a, st);
}

}  // namespace nc
