// fp16 path kernels (fp16 storage, fp32 MFMA accumulation) for gfx950.
//
// k_pw_f16      pointwise / patch-embed / 2x2-s2 / upsample / reconstruction
//               contractions (out^T = W * act^T + b) with gather-on-load and
//               scatter-on-store, and the prior head with the quantiser and
//               the bit partial sums as its epilogue (Fig. 4 "Q", Supp. B.2).
// k_dcblock_f16 one whole DC block (Supp. B.1): depthwise 3x3, pw C->2C +
//               LeakyReLU chained into pw 2C->C through registers 32 hidden
//               channels at a time, residual add; or the gated form (WSiLU
//               and Chunk, pw C->C) with the same pipeline.
#include "common.hpp"
#include "internal.hpp"

#include <cstring>
#include <type_traits>
#include <utility>

namespace nc {

// f(integral_constant<int, T>) for every T of the sequence, in order
template <typename F, int... T>
__device__ __forceinline__ void unrolled_steps(F& f, std::integer_sequence<int, T...>) {
  (f(std::integral_constant<int, T>{}), ...);
}

// ---------------------------------------------------------------- pointwise
// out^T[rows n0 .. n0+NT)[128 pixels] = W * act^T (+ bias) for one tile of
// 128 consecutive output pixels.  8 waves: wave w owns pixels 32 (w & 3) ..
// +31 and rows (w >> 2) NT/2 .. +NT/2.  K is consumed 64 at a time through three
// LDS stages (distinct objects, statically indexed), each holding the
// activation slice (128 pixels x 64 channels, one 128-byte row per pixel,
// 16-byte vector v of pixel px stored at slot v ^ ((px / 2) & 7), which keeps
// the 16 lanes of each quarter of a B-fragment read on distinct banks) and the weight
// fragments of those 64 contraction indices, filled by direct global->LDS
// loads two stages ahead.  Three stages leave room for two workgroups per CU,
// so one workgroup's load latency and stores overlap the other's MFMA work.
// The result is parked in LDS and written with coalesced 16-byte stores.
template <int NT>
struct PwSmem {
  static constexpr int ACT = 128 * 128;               // activation slice bytes
  static constexpr int WGT = NT / 32 * 4 * 1024;      // weight fragments bytes
  static constexpr int STAGE = ACT + WGT;
  static constexpr int DMA_PER_WAVE = (ACT / 1024 + WGT / 1024) / 8;
};

// Global address of 16-byte activation vector v (8 contraction indices
// starting at 64 kc + 8 v) of output pixel gp; n0 = the first output row of
// the workgroup's pass.
template <int LOADER>
__device__ __forceinline__ const char* pw_act_src(const PwArgs& a, int gp, int kc, int v, int n0) {
  const int k = 64 * kc + 8 * v;
  if constexpr (LOADER == LD_NHWC) {
    if (k < a.C0) return (const char*)((const f16*)a.src0 + (size_t)gp * (a.ld0 ? a.ld0 : a.C0) + k);
    return (const char*)((const f16*)a.src1 + (size_t)gp * a.C1 + (k - a.C0));
  } else if constexpr (LOADER == LD_FRAME || LOADER == LD_FRAME_CTX) {
    if (LOADER == LD_FRAME_CTX && kc >= 3) return (const char*)((const f16*)a.src1 + (size_t)gp * a.C1 + (k - 192));
    // unshuffle x8: k = 64 c + 8 i + j -> colour c = kc, frame row 8 py + i = 8 py + v, columns 8 px .. +7
    const int py = gp / a.w8, px = gp - py * a.w8;
    return (const char*)((const f16*)a.src0 + (size_t)kc * a.H * a.W + (size_t)(8 * py + v) * a.W + 8 * px);
  } else if constexpr (LOADER == LD_UP_CTX) {
    if (k < a.C0) return (const char*)((const f16*)a.src0 + (size_t)gp * a.C0 + k);
    const int sp = n0 / a.Cdst, w16 = a.w8 >> 1;
    const int Y = gp / w16, X = gp - Y * w16;
    const int child = (2 * Y + (sp >> 1)) * a.w8 + 2 * X + (sp & 1);
    return (const char*)((const f16*)a.src1 + (size_t)child * a.C1 + (k - a.C0));
  } else {
    // 2x2 stride 2: k = (2 i + j) Csrc + c from pixel (2 Y + i, 2 X + j)
    const int w16 = a.w8 >> 1;
    const int Y = gp / w16, X = gp - Y * w16;
    const int tap = k / a.Csrc, c = k - tap * a.Csrc;
    const int pix = (2 * Y + (tap >> 1)) * a.w8 + 2 * X + (tap & 1);
    return (const char*)((const f16*)a.src0 + (size_t)pix * a.Csrc + c);
  }
}

template <int NT, int LOADER>
__device__ __forceinline__ void pw_issue(const PwArgs& a, int tile, int n0, int kc, char* stage, int wave, int lane) {
  using S = PwSmem<NT>;
  constexpr int ACT_INSTR = S::ACT / 1024;  // 16
#pragma unroll
  for (int i = 0; i < ACT_INSTR / 8; ++i) {
    const int ins = wave + 8 * i;
    const int slot = ins * 64 + lane;
    const int px = slot >> 3, v = (slot & 7) ^ ((px >> 1) & 7);
    const int gp = min(tile * 128 + px, a.P - 1);  // pixels past the end reload the last one
    dma16(pw_act_src<LOADER>(a, gp, kc, v, n0), stage + ins * 1024);
  }
  const int ks = a.K / 16;
  const char* w = (const char*)a.wfrag;
#pragma unroll
  for (int i = 0; i < S::WGT / 1024 / 8; ++i) {
    const int f = wave + 8 * i;  // fragment f of the stage: row tile f / 4, k-step f % 4
    const int mt = n0 / 32 + (f >> 2), sk = 4 * kc + (f & 3);
    dma16(w + (((size_t)mt * ks + sk) * 64 + lane) * 16, stage + S::ACT + f * 1024);
  }
}

template <int NT>
__device__ __forceinline__ void pw_compute(const char* stage, int pg, int hf, int lane, floatx16* acc) {
  using S = PwSmem<NT>;
  constexpr int RT = NT / 64;  // row tiles per wave
  const int pl = pg * 32 + (lane & 31), h = lane >> 5;
  half8 b[4];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) b[ks] = *(const half8*)(stage + pl * 128 + ((((2 * ks + h) ^ ((pl >> 1) & 7))) << 4));
  half8 w[RT][4];
#pragma unroll
  for (int t = 0; t < RT; ++t)
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) w[t][ks] = *(const half8*)(stage + S::ACT + ((hf * RT + t) * 4 + ks) * 1024 + lane * 16);
#pragma unroll
  for (int ks = 0; ks < 4; ++ks)
#pragma unroll
    for (int t = 0; t < RT; ++t) acc[t] = mfma_f16(w[t][ks], b[ks], acc[t]);
}

template <int NT, int LOADER, int EPI>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(NT == 64 ? 4 : 2))) void k_pw_f16(PwArgs a) {
  using S = PwSmem<NT>;
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

  floatx16 acc[RT];
#pragma unroll
  for (int t = 0; t < RT; ++t) acc[t] = floatx16{};
  floatx4 bias[RT][4];
#pragma unroll
  for (int t = 0; t < RT; ++t)
#pragma unroll
    for (int g = 0; g < 4; ++g) bias[t][g] = *(const floatx4*)((const float*)a.bias + n0 + 32 * (hf * RT + t) + 8 * g + 4 * h);

  pw_issue<NT, LOADER>(a, tile, n0, 0, st0, wave, lane);
  if (nk > 1) pw_issue<NT, LOADER>(a, tile, n0, 1, st1, wave, lane);
  // Stage kc: wait until at most the later-issued stages are in flight, make
  // every wave's loads visible, refill the buffer freed in the previous
  // iteration with stage kc + 3, then compute.
  auto step = [&](int kc, const char* cur, char* refill) {
    const int ahead = min(nk - 1 - kc, 1);  // stages issued after kc still in flight
    if (ahead == 1) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(S::DMA_PER_WAVE) : "memory");
    else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    lds_barrier();
    if (kc + 2 < nk) pw_issue<NT, LOADER>(a, tile, n0, kc + 2, refill, wave, lane);
    pw_compute<NT>(cur, pg, hf, lane, acc);
  };
  for (int kc = 0; kc < nk; kc += 3) {
    step(kc, st0, st2);
    if (kc + 1 < nk) step(kc + 1, st1, st0);
    if (kc + 2 < nk) step(kc + 2, st2, st1);
  }
  lds_barrier();  // every wave is done reading the stages

  // park acc + bias as fp32, one row of NT floats per tile pixel, 16-byte
  // chunk c of the row of pixel px at c ^ (px & SWZ); the 128 rows fill the
  // stage buffers in order, RPB rows per buffer
  constexpr int SWZ = (NT / 4 - 1) & 31;
  constexpr int ROW = NT * 4, RPB = S::STAGE / ROW;
  static_assert(3 * RPB >= 128, "the tile's rows fit three stage buffers");
  auto park_row = [&](int px) __attribute__((always_inline)) -> char* {
    const int b = px / RPB, r = px - b * RPB;
    return (b == 0 ? st0 : b == 1 ? st1 : st2) + r * ROW;
  };
  {
    const int row = lane & 31;
    char* ob = park_row(32 * pg + row);
#pragma unroll
    for (int t = 0; t < RT; ++t)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int nl = 32 * (hf * RT + t) + 8 * g + 4 * h;  // row of the pass
        floatx4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = acc[t][4 * g + e] + bias[t][g][e];
        *(floatx4*)(ob + (((nl >> 2) ^ (row & SWZ)) << 4)) = o;
      }
  }
  // prior head: a pass covers channels c0 .. c0+31 (rows 0-31 mu, 32-63 s);
  // the tile's symbols are staged in stage buffer 2 as [channel][pixel]
  const int c0 = a.c_off + n0 / 2;
  int16_t* qt = (int16_t*)st2;
  uint8_t* kt = (uint8_t*)(st2 + 8192);  // scale indices, [channel][pixel]
  float* sct = (float*)(st2 + 12288);    // the coder scales, for the scale-index search
  if constexpr (EPI == EP_SCALES || EPI == EP_PRIOR) {
    if (threadIdx.x < kCoderScales && a.k_out) sct[threadIdx.x] = a.scales[threadIdx.x];
  }
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
    const int ch = threadIdx.x >> 4, k = threadIdx.x & 15;  // 32 channels x 16 chunks of 8 pixels
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

  auto parked = [&](int px, int nl8) {  // 8 floats: pass rows nl8 * 8 .. +7 of tile pixel px
    const int row = px & 31;
    const char* ob = park_row(px);
    const floatx4 o0 = *(const floatx4*)(ob + (((2 * nl8) ^ (row & SWZ)) << 4));
    const floatx4 o1 = *(const floatx4*)(ob + (((2 * nl8 + 1) ^ (row & SWZ)) << 4));
    floatx16 r;  // only [0, 8) used
#pragma unroll
    for (int e = 0; e < 4; ++e) { r[e] = o0[e]; r[4 + e] = o1[e]; }
    return r;
  };
  // (mu, s) of 8 channels c .. c + 7 of pixel gp: the head's rows plus the
  // addend of the two-step entropy model (hyper parameters, or the first
  // step's (mu, s) for the second step)
  auto prior_ms = [&](int px, int g8, int gp, float* mu, float* sg) __attribute__((always_inline)) {
    const floatx16 m = parked(px, g8), sv = parked(px, 4 + g8);
#pragma unroll
    for (int e = 0; e < 8; ++e) { mu[e] = m[e]; sg[e] = sv[e]; }
    if (a.add && gp < a.P) {
      const size_t at = (size_t)gp * a.add_ld + (c0 + 8 * g8 - a.add_c0);
      if (a.add_f32) {
        const float* am = (const float*)a.add + at;
#pragma unroll
        for (int e = 0; e < 8; ++e) { mu[e] += am[e]; sg[e] += am[a.add_s + e]; }
      } else {
        const half8 hm = *(const half8*)((const f16*)a.add + at), hs = *(const half8*)((const f16*)a.add + at + a.add_s);
#pragma unroll
        for (int e = 0; e < 8; ++e) { mu[e] += (float)hm[e]; sg[e] += (float)hs[e]; }
      }
    }
  };
  // channels >= split: (mu, s) go to the base buffer for the second step
  const bool to_base = a.split && c0 >= a.split;
  auto store_base = [&](int g8, int gp, const float* mu, const float* sg) __attribute__((always_inline)) {
    if (gp >= a.P) return;
    const int nb = a.Cdst - a.split;
    float* b = (float*)a.base + (size_t)gp * 2 * nb + (c0 + 8 * g8 - a.split);
    *(floatx4*)b = floatx4{mu[0], mu[1], mu[2], mu[3]};
    *(floatx4*)(b + 4) = floatx4{mu[4], mu[5], mu[6], mu[7]};
    *(floatx4*)(b + nb) = floatx4{sg[0], sg[1], sg[2], sg[3]};
    *(floatx4*)(b + nb + 4) = floatx4{sg[4], sg[5], sg[6], sg[7]};
  };
  if constexpr (EPI == EP_SCALES) {
    const int px = threadIdx.x >> 2, g8 = threadIdx.x & 3;
    const int gp = tile * 128 + px;
    float mu[8], sg[8];
    prior_ms(px, g8, gp, mu, sg);
    if (to_base) {
      store_base(g8, gp, mu, sg);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) kt[(8 * g8 + e) * 128 + px] = (uint8_t)coder_scale_index(softplus_sigma(sg[e]), sct);
      // mu as fp32 (NHWC), for yhat = q + mu once the symbols are decoded
      if (a.dst && gp < a.P) {
        float* dm = (float*)a.dst + (size_t)gp * a.Cdst + c0 + 8 * g8;
        *(floatx4*)dm = floatx4{mu[0], mu[1], mu[2], mu[3]};
        *(floatx4*)(dm + 4) = floatx4{mu[4], mu[5], mu[6], mu[7]};
      }
    }
    lds_barrier();
    if (!to_base) store_k();
  } else if constexpr (EPI == EP_PRIOR || EPI == EP_PRIOR_DEC) {
    // thread = (pixel px, 8 channels g8): mu and s from the park, y / q, yhat
    const int px = threadIdx.x >> 2, g8 = threadIdx.x & 3;
    const int gp = tile * 128 + px;
    const int c = c0 + 8 * g8;
    float mu[8], sg[8];
    prior_ms(px, g8, gp, mu, sg);
    double bsum = 0.0;
    if (to_base) {
      store_base(g8, gp, mu, sg);
      if constexpr (EPI == EP_PRIOR)
        if (threadIdx.x == 0) a.partials[(size_t)tile * npass + n0 / NT] = 0.0;
    } else if constexpr (EPI == EP_PRIOR) {
      if (a.k_out) {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          kt[(8 * g8 + e) * 128 + px] = (uint8_t)coder_scale_index(softplus_sigma(sg[e]), sct);
      }
      half8 yv = {};
      if (gp < a.P) yv = *(const half8*)((const f16*)a.y + (size_t)gp * a.Cdst + c);
      half8 yh;
      float b8 = 0.f;  // the thread's 8 symbols in fp32, then the fixed-order double sums
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float q = rintf((float)yv[e] - mu[e]);
        q = fminf(fmaxf(q, -32768.f), 32767.f);
        qt[(8 * g8 + e) * 128 + px] = (int16_t)q;
        yh[e] = (f16)(q + mu[e]);
        b8 += symbol_bits(q, softplus_sigma(sg[e]));
      }
      if (gp < a.P) bsum = (double)b8;
      if (gp < a.P) *(half8*)((f16*)a.dst + (size_t)gp * a.Cdst + c) = yh;
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
        half8 yh;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          // same operation order as the encoder: mu first, then q + mu
          const float q = (float)qt[(8 * g8 + e) * 128 + px];
          yh[e] = (f16)(q + mu[e]);
        }
        *(half8*)((f16*)a.dst + (size_t)gp * a.Cdst + c) = yh;
      }
    }
  } else if constexpr (EPI == EP_ZQUANT) {
    // the 64 rows are the channels of z: q_z = round(z) (staged [channel][pixel]
    // in stage buffer 2, 16 KiB), zhat = q_z (NHWC), rate under sigma_z[c]
    static_assert(NT == 64, "z has 64 channels");
    const int px = threadIdx.x >> 2, g8 = threadIdx.x & 3;
    const int gp = tile * 128 + px;
    double bsum = 0.0;
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      const int cz = 32 * half + 8 * g8;
      const floatx16 zv = parked(px, 4 * half + g8);
      half8 zh;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float q = rintf(zv[e]);
        q = fminf(fmaxf(q, -32768.f), 32767.f);
        qt[(cz + e) * 128 + px] = (int16_t)q;
        zh[e] = (f16)q;
        if (gp < a.P) bsum += (double)symbol_bits(q, a.zsigma[cz + e]);
      }
      if (gp < a.P) *(half8*)((f16*)a.dst + (size_t)gp * a.Cdst + cz) = zh;
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
    // rows 64 j .. 64 j + 31 of the pass are h1 of gated channels n0 / 2 + 32 j
    // .. + 31, rows 64 j + 32 .. + 63 the matching h2 (the packed pw1 order).
    // As the fused gated block: WSiLU(h1) = h1 sigmoid(4 h1) rounded to fp16,
    // then g = WSiLU(h1) h2 rounded to fp16.
    constexpr int G = NT / 64, GU = 128 * G * 4;  // units (pixel, group, 8 channels)
#pragma unroll
    for (int it = 0; it < GU / 512; ++it) {
      const int idx = it * 512 + threadIdx.x;
      const int px = idx / (4 * G), j = (idx >> 2) % G, g8 = idx & 3;
      const int gp = tile * 128 + px;
      if (gp < a.P) {
        const floatx16 h1 = parked(px, 8 * j + g8), h2 = parked(px, 8 * j + 4 + g8);
        half8 o;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float u = h1[e];
          const f16 s1 = (f16)(u / (1.f + __expf(-4.f * u)));
          o[e] = (f16)((float)s1 * h2[e]);
        }
        *(half8*)((f16*)a.dst + (size_t)gp * a.Cdst + n0 / 2 + 32 * j + 8 * g8) = o;
      }
    }
  } else if constexpr (EPI == EP_REC) {
    // rows of the pass: global rows n0 .. n0+NT = 64 c + 8 i + j; a 16-byte store
    // covers the 8 frame pixels j of (colour c, row i) of one 1/8-scale pixel.
    constexpr int UNITS = 128 * (NT / 8);
#pragma unroll
    for (int it = 0; it < UNITS / 512; ++it) {
      const int idx = it * 512 + threadIdx.x;
      const int nl8 = idx >> 7, px = idx & 127;  // consecutive threads walk pixels
      const int gp = tile * 128 + px;
      if (gp < a.P) {
        const floatx16 r = parked(px, nl8);
        const int n = n0 + 8 * nl8, c = n >> 6, i = (n >> 3) & 7;
        const int py = gp / a.w8, pxx = gp - py * a.w8;
        half8 o;
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] = (f16)fminf(fmaxf(r[e], 0.f), 1.f);
        *(half8*)((f16*)a.dst + (size_t)c * a.H * a.W + (size_t)(8 * py + i) * a.W + 8 * pxx) = o;
      }
    }
  } else {
    constexpr int UNITS = 128 * (NT / 8);
#pragma unroll
    for (int it = 0; it < UNITS / 512; ++it) {
      const int idx = it * 512 + threadIdx.x;
      const int px = idx / (NT / 8), nl8 = idx % (NT / 8);  // consecutive threads walk a pixel's row
      const int gp = tile * 128 + px;
      if (gp < a.P) {
        const floatx16 r = parked(px, nl8);
        half8 o;
        if constexpr (EPI == EP_LRELU) {
          // as the fused block: the hidden value rounded to fp16, then
          // max(h, 0.1 h) in fp16
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const f16 hv = (f16)r[e];
            o[e] = __builtin_fmaxf16(hv, hv * (f16)0.1f);
          }
        } else if constexpr (EPI == EP_RESID) {
          const half8 zr = *(const half8*)((const f16*)a.res + (size_t)gp * a.Cdst + n0 + 8 * nl8);
#pragma unroll
          for (int e = 0; e < 8; ++e) o[e] = (f16)(r[e] + (float)zr[e]);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) o[e] = (f16)r[e];
        }
        size_t off;
        if constexpr (EPI == EP_NHWC || EPI == EP_LRELU || EPI == EP_RESID) {
          off = (size_t)gp * a.Cdst + n0 + 8 * nl8;
        } else {  // EP_UP: pass rows n = sp * C + c, all in one sub-position sp
          const int C = a.Cdst, n = n0 + 8 * nl8;
          const int sp = n / C, c = n - sp * C;
          const int w16 = a.w8 >> 1;
          const int Y = gp / w16, X = gp - Y * w16;
          off = (size_t)((2 * Y + (sp >> 1)) * a.w8 + 2 * X + (sp & 1)) * C + c;
        }
        *(half8*)((f16*)a.dst + off) = o;
      }
    }
  }
}

// One DC block (Supp. B.1) for a tile of 128 pixels, 8 waves.
//
// Waves w and w+4 share 32 pixels (pixel group w & 3) and sit on the same
// SIMD; wave w >> 2 == hf owns output channels [hf C/2, (hf+1) C/2) of the
// second pointwise conv and produces the hidden chunks j with j % 2 == hf of
// the first one.  A hidden chunk (32 channels after bias + LeakyReLU, fp16)
// goes to LDS in MFMA operand order so both waves of the pair consume it.
//
// The weights of one block are streamed in NCH = 2C/32 chunks: chunk j holds
// the KS = C/16 pw1 fragments of hidden channels 32 j .. +31, their bias in
// one more fragment (32 fp32 values that start the chain), then the 2 MT
// pw2 fragments that consume them (one 1 KiB MFMA A fragment each), into a
// ring of four LDS buffers with direct global->LDS loads (the loop is unrolled
// by four, so every buffer address is static).  The residual is added from
// LDS in the epilogue, so the prologue only exchanges the filtered channels.
template <int C>
struct DcSmem {
  static constexpr int KS = C / 16, MT = C / 32, FR = KS + 1 + 2 * MT, CHUNK = FR * 1024;
};

// Fragments 0 .. n-1 of chunk j -> buf (n = FR, or KS + 1 for a gated h1
// entry, whose pw2 slots are unused); fragment f is loaded by wave f % 8, so
// every wave issues at least n / 8 loads.
template <int C>
__device__ __forceinline__ void dc_issue(const char* wchunks, int j, char* buf, int wave, int lane, int n) {
  constexpr int FR = DcSmem<C>::FR;
#pragma unroll
  for (int i = 0; i < (FR + 7) / 8; ++i) {
    const int f = wave + 8 * i;
    if (f < n) dma16(wchunks + ((size_t)j * FR + f) * 1024 + lane * 16, buf + f * 1024);
  }
}

// The first half of the pw1 fragments of one chunk, to registers.
template <int C>
__device__ __forceinline__ void dc_load_w1(const char* wb, int lane, half8* wf) {
  const half8* w = (const half8*)wb + lane;
#pragma unroll
  for (int s = 0; s < DcSmem<C>::KS / 2; ++s) wf[s] = w[s * 64];
}

// pw1 chain of one hidden chunk, starting from its bias: the first half of
// the fragments comes from registers (loaded an iteration earlier), the second
// half and the bias are read from the chunk's buffer while the first half runs.
template <int C>
__device__ __forceinline__ floatx16 dc_hidden(const half8* wf, const char* wb, const half8* av, int lane) {
  constexpr int KS = DcSmem<C>::KS;
  const half8* w = (const half8*)wb + lane;
  half8 w2[KS / 2];
#pragma unroll
  for (int s = 0; s < KS / 2; ++s) w2[s] = w[(KS / 2 + s) * 64];
  // the bias: 32 fp32 values at the start of fragment KS; row 8 g + 4 h + e of
  // the accumulator is element 4 g + e of lane half h
  const int h = lane >> 5;
  floatx4 bv[4];
#pragma unroll
  for (int g = 0; g < 4; ++g) bv[g] = *(const floatx4*)(wb + KS * 1024 + (8 * g + 4 * h) * 4);
  __builtin_amdgcn_sched_barrier(0);
  floatx16 hacc;
#pragma unroll
  for (int g = 0; g < 4; ++g)
#pragma unroll
    for (int e = 0; e < 4; ++e) hacc[4 * g + e] = bv[g][e];
#pragma unroll
  for (int s = 0; s < KS / 2; ++s) hacc = mfma_f16(wf[s], av[s], hacc);
#pragma unroll
  for (int s = 0; s < KS / 2; ++s) hacc = mfma_f16(w2[s], av[KS / 2 + s], hacc);
  return hacc;
}

// LeakyReLU, fp16; stored to `gx` as two B fragments (k = hidden in the
// permuted order the pw2 weights were packed with).
__device__ __forceinline__ void dc_hidden_store(const floatx16& hacc, int lane, half8* gx) {
  half8 g0, g1;
#pragma unroll
  for (int g = 0; g < 4; ++g)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const f16 v = (f16)leaky(hacc[4 * g + e]);
      if (g < 2) g0[4 * g + e] = v; else g1[4 * (g - 2) + e] = v;
    }
  gx[lane] = g0;
  gx[64 + lane] = g1;
}

// Gated form.  WSiLU(h1) = h1 sigmoid(4 h1) of the h1 chain, kept as fp16 (8
// registers) until the pair's h2 chain is done; then g = WSiLU(h1) * h2 for
// the same elements, fp16, stored like dc_hidden_store.
struct Wsilu16 {
  half8 v[2];
};
__device__ __forceinline__ Wsilu16 dc_wsilu(const floatx16& h1) {
  Wsilu16 w;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const float u = h1[r];
    w.v[r >> 3][r & 7] = (f16)(u / (1.f + __expf(-4.f * u)));
  }
  return w;
}
__device__ __forceinline__ void dc_gate_store(const Wsilu16& s1, const floatx16& h2, int lane, half8* gx) {
  half8 g0, g1;
#pragma unroll
  for (int g = 0; g < 4; ++g)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int r = 4 * g + e;
      const f16 v = (f16)((float)s1.v[r >> 3][r & 7] * h2[r]);
      if (g < 2) g0[4 * g + e] = v; else g1[4 * (g - 2) + e] = v;
    }
  gx[lane] = g0;
  gx[64 + lane] = g1;
}

// Second pointwise conv, hidden chunk j, this wave's MT/2 output tiles.
template <int C>
__device__ __forceinline__ void dc_project(const char* wb, const half8* gx, int hf, int lane, floatx16* out) {
  constexpr int KS = DcSmem<C>::KS, MT = DcSmem<C>::MT;
  const half8* w = (const half8*)wb + lane;
  const half8 g0 = gx[lane], g1 = gx[64 + lane];
#pragma unroll
  for (int t = 0; t < MT / 2; ++t) {
    const int tt = hf * (MT / 2) + t;
    out[t] = mfma_f16(w[(KS + 1 + 2 * tt) * 64], g0, out[t]);
    out[t] = mfma_f16(w[(KS + 1 + 2 * tt + 1) * 64], g1, out[t]);
  }
}

// Depthwise geometry of the DC block for C channels.  Wave w filters NCW
// channels (block w % NCB) over NRW tile rows (block w / NCB); lane = channel
// pair cp (fastest) x column slice colq of CPL columns, so each lane keeps its
// 9 tap weights in registers and slides a 3 x 3 window over its columns.  The
// wave's halo band ((NRW + 2) x 18 pixels x NCW channels) sits in its own LDS
// region: halo pixel hp at position hp ^ ((hp >> 2) & 1), which puts the
// pixels read by the column slices of one half-wave in different banks when
// a pixel's slice is shorter than 128 bytes.  With C = 256 a wave takes 64
// channels (whole 128-byte lines per halo pixel for its direct loads).
template <int C>
struct DcDw {
  static constexpr int NCW = C == 256 ? 64 : C >= 128 ? C / 8 : 16;  // channels per wave
  static constexpr int NRW = C / NCW;                 // tile rows per wave
  static constexpr int NCB = C / NCW;                 // channel blocks
  static constexpr int NCP = NCW / 2;                 // channel pairs
  static constexpr int NCOLQ = 64 / NCP;              // column slices
  static constexpr int CPL = 16 / NCOLQ;              // columns per lane
  static constexpr int BP = (NRW + 2) * 18;           // halo pixels of the band
  static constexpr int UPP = NCW / 8;                 // 16-byte units per halo pixel
  static constexpr int SLOTS = BP * UPP;
  static constexpr int RINSTR = (SLOTS + 63) / 64;    // direct loads per wave for the band
  static constexpr int RB = SLOTS * 16;               // region bytes
  static constexpr int XF = 1024 + 16;                // exchange fragment stride (padded against bank conflicts)
  static constexpr int SPW = NCW / 16;                // 16-channel MFMA steps per wave
  static_assert(NCB * (8 / NRW) == 8 && NCOLQ * CPL == 16 && BP % 2 == 0 && NRW % 2 == 0, "C in {64, 128, 256}");
  static_assert(SPW * (NRW / 2) * XF <= RB, "the exchange fits the band's region");
};

__device__ __forceinline__ int dw_pos(int hp) { return hp ^ ((hp >> 2) & 1); }

// GATED: the gated form (Supp. B.1, WSiLU and Chunk).  The weight entries
// alternate: entry 2p holds the pw1 fragments and bias of h1 rows 32 p .. +31,
// entry 2p + 1 those of the matching h2 rows and the pw2 fragments of gated
// channels 32 p .. +31.  One wave produces both chains of pair p (wave p % 2
// of its SIMD pair), keeps h1 in registers, and gates when h2 is done; the
// pair is projected in the next iteration (odd entries), so even iterations
// run no pw2.
template <int C, bool GATED>
__global__ __launch_bounds__(512) void k_dcblock_f16(BlockArgs a) {
  using G = DcDw<C>;
  constexpr int KS = DcSmem<C>::KS;
  constexpr int NCH = 2 * C / 32;  // hidden chunks of 32 (a multiple of 4)
  constexpr int MT = DcSmem<C>::MT;
  constexpr int FR = DcSmem<C>::FR;
  constexpr int TH = 8, TW = 16;   // pixel tile (rows x columns at 1/8 scale)
  constexpr int CH8 = C / 8;       // 16-byte channel vectors per pixel
  static_assert(NCH % 4 == 0, "chunk loop is unrolled by four");
  // LDS: chunk buffers 0-3, the hidden-chunk buffers, the pw2 bias.  The
  // eight band regions start after the pw1 part (fragments 0 .. KS) of buffer
  // 1 and are laid over the rest, which is dead once the filtered channels have
  // been exchanged.  So chunk 0 and the pw1 part of chunk 1 are loaded from
  // the start, the pw2 part of chunk 1 after the exchange.  After the loop
  // buffers 0-1 hold the residual tile and buffers 2-3 the parked output.
  constexpr int BUF = DcSmem<C>::CHUNK;
  constexpr int O1 = BUF, O2 = 2 * BUF, O3 = 3 * BUF, OGX = 4 * BUF;
  constexpr int OR = BUF + (KS + 1) * 1024;  // first band region
  constexpr int OB2 = (OR + 8 * G::RB > OGX + 16384 ? OR + 8 * G::RB : OGX + 16384);  // pw2 bias (C fp32)
  constexpr int SMEM = OB2 + 1024;
  static_assert(SMEM <= 160 * 1024, "fits the LDS of a CU");
  static_assert(128 * C * 2 <= 2 * BUF && 2 * 32 * C * 2 <= BUF && BUF % 1024 == 0, "residual tile and parked output fit");
  __shared__ __attribute__((aligned(1024))) char smem[SMEM];
  char* const wb0 = smem;
  char* const wb1 = smem + O1;
  char* const wb2 = smem + O2;
  char* const wb3 = smem + O3;
  half8* const gx0 = (half8*)(smem + OGX);         // [pixel group][2 fragments x 64 lanes], even chunks
  half8* const gx1 = (half8*)(smem + OGX + 8192);  // odd chunks

  const int tiles_x = (a.w + TW - 1) / TW;
  const int ntile = tiles_x * ((a.h + TH - 1) / TH);
  const int tile = xcd_tile(blockIdx.x, gridDim.x);
  if (tile >= ntile) return;
  const int ty0 = (tile / tiles_x) * TH, tx0 = (tile % tiles_x) * TW;
  const int lane = threadIdx.x & 63, h = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int pg = wave & 3, hf = wave >> 2;  // MFMA role: 32 pixels, half the outputs
  const f16* z = (const f16*)a.src;
  const char* wchunks = (const char*)a.w1;
  auto region = [&](int w_) __attribute__((always_inline)) -> char* { return smem + OR + w_ * G::RB; };

  // Depthwise role.
  const int cbk = wave % G::NCB, rbk = wave / G::NCB;
  const int cp = lane % G::NCP, colq = lane / G::NCP;
  const int c0 = cbk * G::NCW + 2 * cp;  // this lane's channels c0, c0 + 1
  char* const own = region(wave);
  // this pair's 9 taps (fp16 pairs) and two fp32 biases: 48 bytes per pair
  half2 wt[9];
  float bias0, bias1;
  {
    // 11 words: a loaded word left unused would be reused as a temporary by
    // the compiler, which then waits for this load before the band is issued
    const intx4* wsrc = (const intx4*)a.dww + 3 * (c0 / 2);
    const intx4 q0 = wsrc[0], q1 = wsrc[1];
    const intx3 q2 = *(const intx3*)(wsrc + 2);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int x0 = q0[i], x1 = q1[i];
      wt[i] = __builtin_bit_cast(half2, x0);
      wt[4 + i] = __builtin_bit_cast(half2, x1);
    }
    const int x8 = q2[0], xb0 = q2[1], xb1 = q2[2];
    wt[8] = __builtin_bit_cast(half2, x8);
    bias0 = __builtin_bit_cast(float, xb0);
    bias1 = __builtin_bit_cast(float, xb1);
  }
  // pw2 bias to LDS (wave 0, before its band: waited for with the band)
  if (wave == 0 && lane < C / 4) dma16((const float*)a.b2 + 4 * lane, smem + OB2);
  // Halo band: slot S = 16-byte unit S of the region holds unit S % UPP of
  // halo pixel dw_pos(S / UPP); out-of-image pixels read the zero row.
#pragma unroll
  for (int i = 0; i < G::RINSTR; ++i) {
    const int S = i * 64 + lane;
    if (G::SLOTS % 64 == 0 || S < G::SLOTS) {
      const int hp = dw_pos(S / G::UPP), u = S % G::UPP;
      const int hy = ty0 + rbk * G::NRW - 1 + hp / 18, hx = tx0 - 1 + hp % 18;
      const bool in = hy >= 0 && hy < a.h && hx >= 0 && hx < a.w;
      dma16(in ? z + (size_t)(hy * a.w + hx) * C + cbk * G::NCW + 8 * u : (const f16*)a.zpad, own + i * 1024);
    }
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this wave's band

  // Chunk 0 and the pw1 part of chunk 1 (consumed after the depthwise) are
  // requested a few fragments per output row, so that their direct loads,
  // which the memory pipeline takes one at a time, queue behind the band
  // instead of ahead of it.  Load m < NP0 is fragment wave + 8 m of chunk 0,
  // the others fragment wave + 8 (m - NP0) of chunk 1.
  constexpr int NP0 = (FR + 7) / 8, NP1 = (KS + 1 + 7) / 8;
  constexpr int PER_ROW = (NP0 + NP1 + G::NRW - 1) / G::NRW;
  auto issue_early = [&](int n) __attribute__((always_inline)) {
#pragma unroll
    for (int m = n * PER_ROW; m < (n + 1) * PER_ROW && m < NP0 + NP1; ++m) {
      const int c1 = m >= NP0;
      const int f = wave + 8 * (c1 ? m - NP0 : m);
      if (f < (c1 ? KS + 1 : FR))
        dma16(wchunks + ((size_t)c1 * FR + f) * 1024 + lane * 16, (c1 ? wb1 : wb0) + f * 1024);
    }
  };
  // Depthwise 3x3 + bias: every band value this lane needs first, then the
  // sliding window (fp32 accumulation), rounded to fp16.
  half2 v[G::NRW + 2][G::CPL + 2];
#pragma unroll
  for (int y = 0; y < G::NRW + 2; ++y)
#pragma unroll
    for (int x = 0; x < G::CPL + 2; ++x)
      v[y][x] = *(const half2*)(own + dw_pos(y * 18 + colq * G::CPL + x) * (G::UPP * 16) + cp * 4);
  // The filtered pair goes straight to the MFMA B fragment of its pixel group
  // and 16-channel step, in this wave's region (the band is dead once read):
  // fragment (row pair j, step i) at (j SPW + i) XF; lane (pixel & 31) +
  // 32 (bit 3 of the channel), element channel & 7.
  const int xhalf = (cp >> 2) & 1;
#pragma unroll
  for (int rr = 0; rr < G::NRW; ++rr)
#pragma unroll
    for (int k = 0; k < G::CPL; ++k) {
      float a0 = bias0, a1 = bias1;
#pragma unroll
      for (int ky = 0; ky < 3; ++ky)
#pragma unroll
        for (int kx = 0; kx < 3; ++kx) {
          const half2 zz = v[rr + ky][k + kx], ww = wt[3 * ky + kx];
          a0 = fmaf((float)ww[0], (float)zz[0], a0);
          a1 = fmaf((float)ww[1], (float)zz[1], a1);
        }
      half2 o;
      o[0] = (f16)a0;
      o[1] = (f16)a1;
      const int px = 16 * (rr & 1) + colq * G::CPL + k;  // pixel within the 32-pixel group
      const int f = (rr >> 1) * G::SPW + (cp >> 3);
      *(half2*)(own + f * G::XF + (px + 32 * xhalf) * 16 + (cp & 3) * 4) = o;
      if (k == G::CPL - 1) issue_early(rr);
    }
  lds_barrier();

  // MFMA role: all C filtered channels of this wave's 32 pixels.
  half8 av[KS];
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    const int wcb = s / G::SPW, wrb = (2 * pg) / G::NRW;  // writer wave's channel and row blocks
    const int f = (pg - wrb * (G::NRW / 2)) * G::SPW + (s - wcb * G::SPW);
    av[s] = *(const half8*)(region(wrb * G::NCB + wcb) + f * G::XF + lane * 16);
  }
  lds_barrier();  // exchange read: the regions take buffers 2, 3 and the hidden chunks from here on

  // Pipeline: in iteration j one wave of each pair runs the pw1 chain of
  // hidden chunk j+1 from fragments it loaded in iteration j-1, the other loads
  // the fragments of chunk j+2 for its next chain; both project hidden chunk
  // j.  Chunk c sits in buffer c % 4; chunk j+3 is loaded during iteration j.
  // Chunk 2 is only needed from iteration 1 on: it arrives during hidden
  // chunk 0 and iteration 0, whose chain for chunk 2 loads its own fragments.
  // the pw2 part of chunk 1 (2 MT fragments), then chunk 2
#pragma unroll
  for (int i = 0; i < (2 * MT + 7) / 8; ++i) {
    const int f = KS + 1 + wave + 8 * i;
    if ((2 * MT) % 8 == 0 || f < FR) dma16(wchunks + ((size_t)FR + f) * 1024 + lane * 16, wb1 + f * 1024);
  }
  dc_issue<C>(wchunks, 2, wb2, wave, lane, GATED ? KS + 1 : FR);  // gated: chunk 2 is an h1 entry
  half8 wf[KS / 2];  // first half of the next chain's pw1 fragments
  // chunk 0 and the pw1 part of chunk 1 (the rest of chunk 1 and chunk 2 in flight)
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * MT / 8 + (GATED ? KS + 1 : FR) / 8) : "memory");
  lds_barrier();  // chunks 0 and 1 staged
  Wsilu16 sw1 = {};  // gated: WSiLU of the h1 chain of the pair being produced
  if (hf == 0) {
    dc_load_w1<C>(wb0, lane, wf);
    if constexpr (GATED) sw1 = dc_wsilu(dc_hidden<C>(wf, wb0, av, lane));
    else dc_hidden_store(dc_hidden<C>(wf, wb0, av, lane), lane, gx0 + 128 * pg);
  }
  floatx16 out[MT / 2];  // pw2 accumulators, starting from the bias
#pragma unroll
  for (int t = 0; t < MT / 2; ++t) {
    const int tt = hf * (MT / 2) + t;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const floatx4 bv = *(const floatx4*)(smem + OB2 + (32 * tt + 8 * g + 4 * h) * 4);
#pragma unroll
      for (int e = 0; e < 4; ++e) out[t][4 * g + e] = bv[e];
    }
  }
  if (hf == (GATED ? 0 : 1)) dc_load_w1<C>(wb1, lane, wf);  // chunk 1, for its chain in iteration 0
  lds_barrier();  // hidden chunk 0 visible

  // The residual tile (128 pixels x C fp16; 16-byte unit u of pixel px holds
  // channel vector u ^ (px & 7); byte b of the tile in buffer 0 below BUF, in
  // buffer 1 above) is loaded during the last two chunks.
  auto rtile = [&](int b) __attribute__((always_inline)) -> char* { return b < BUF ? wb0 + b : wb1 + (b - BUF); };
  auto issue_residual = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < C / 32; ++i) {
      const int k = wave + 8 * i;  // 1 KiB unit k of the tile
      const int S = k * 64 + lane;
      const int px = S / CH8, k8 = (S % CH8) ^ (px & 7);
      const int yy = ty0 + (px >> 4), xx = tx0 + (px & 15);
      const bool in = yy < a.h && xx < a.w;
      dma16(in ? z + (size_t)(yy * a.w + xx) * C + 8 * k8 : (const f16*)a.zpad, rtile(k * 1024));
    }
  };
  auto step = [&](int j, const char* wcur, const char* wnxt, const char* wpre, char* wiss, half8* gcur, half8* gnxt)
                  __attribute__((always_inline)) {
    const bool dma = j + 3 < NCH;
    if (dma) dc_issue<C>(wchunks, j + 3, wiss, wave, lane, GATED && !((j + 3) & 1) ? KS + 1 : FR);
    // producer of chunk c: wave c % 2 of the pair, or in the gated form (c / 2) % 2
    const int pj1 = GATED ? ((j + 1) >> 1) & 1 : (j + 1) & 1, pj2 = GATED ? ((j + 2) >> 1) & 1 : j & 1;
    const bool produce = j + 1 < NCH && hf == pj1;
    const bool prefetch = j >= 1 && j + 2 < NCH && hf == pj2;
    floatx16 hacc;
    if (produce) {
      // the producer's chain is the iteration's critical path: its MFMAs go
      // first on the SIMD, the partner's projection fills the gaps
      __builtin_amdgcn_s_setprio(2);
      if (j == 1) dc_load_w1<C>(wnxt, lane, wf);  // iteration 0 had no prefetch
      hacc = dc_hidden<C>(wf, wnxt, av, lane);
    }
    if (j == NCH - 2) issue_residual();  // buffers 0 and 1 are free from here on
    if (!GATED || (j & 1)) dc_project<C>(wcur, gcur, hf, lane, out);
    if (prefetch) dc_load_w1<C>(wpre, lane, wf);
    if (produce) {
      if constexpr (GATED) {
        if ((j + 1) & 1) dc_gate_store(sw1, hacc, lane, gnxt);  // h2 of the pair: gate it
        else sw1 = dc_wsilu(hacc);
      } else {
        dc_hidden_store(hacc, lane, gnxt);
      }
    }
    // chunk j+3 (in iteration 0 also chunk 2), or the residual in the last step
    if (dma || j == NCH - 1) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_setprio(0);
    lds_barrier();
  };
  for (int j = 0; j < NCH; j += 4) {
    step(j + 0, wb0, wb1, wb2, wb3, gx0 + 128 * pg, gx1 + 128 * pg);
    step(j + 1, wb1, wb2, wb3, wb0, gx1 + 128 * pg, gx0 + 128 * pg);
    step(j + 2, wb2, wb3, wb0, wb1, gx0 + 128 * pg, gx1 + 128 * pg);
    step(j + 3, wb3, wb0, wb1, wb2, gx1 + 128 * pg, gx0 + 128 * pg);
  }

  // Epilogue.  The residual enters the accumulators through the MFMA: for
  // output tile tt, out += E0 z[32 tt .. +15] + E1 z[32 tt + 16 .. +31] with
  // E0, E1 the two 32 x 16 halves of the identity (exact in fp32), the z
  // fragments read from the residual tile in B layout.  Then the sums are
  // rounded once to fp16 and parked in buffers 2 (pixel groups 0, 1) and 3
  // (groups 2, 3), row = pixel, 8-byte unit u of the row at u ^ (row & 15);
  // each thread finally stores 8 channels of one pixel with one 16-byte store.
  {
    const int row = lane & 31, px = 32 * pg + row;
    half8 e0, e1;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      e0[e] = (f16)(row == 8 * h + e ? 1.f : 0.f);
      e1[e] = (f16)(row == 16 + 8 * h + e ? 1.f : 0.f);
    }
#pragma unroll
    for (int t = 0; t < MT / 2; ++t) {
      const int tt = hf * (MT / 2) + t;
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const int k8 = 4 * tt + 2 * q + h;
        const half8 zb = *(const half8*)rtile((px * CH8 + (k8 ^ (px & 7))) * 16);
        out[t] = mfma_f16(q ? e1 : e0, zb, out[t]);
      }
    }
    char* ob = (pg < 2 ? wb2 : wb3) + (pg & 1) * (32 * C * 2);
#pragma unroll
    for (int t = 0; t < MT / 2; ++t)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int cc = 32 * (hf * (MT / 2) + t) + 8 * g + 4 * h;
        half4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = (f16)out[t][4 * g + e];
        *(half4*)(ob + row * (C * 2) + (((cc >> 2) ^ (row & 15)) << 3)) = o;
      }
  }
  lds_barrier();
  constexpr int PER = 128 * CH8 / 512;  // 16-byte units per thread
  f16* dst = (f16*)a.dst;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int idx = i * 512 + threadIdx.x;
    const int px = idx / CH8, k8 = idx % CH8;
    const int row = px & 31;
    const int yy = ty0 + (px >> 4), xx = tx0 + (px & 15);
    if (yy < a.h && xx < a.w) {
      // units 2 k8 and 2 k8 + 1 are the aligned pair at 2 k8 ^ (row & 14),
      // in swapped order when row is odd
      const char* ob = (px < 64 ? wb2 : wb3) + ((px >> 5) & 1) * (32 * C * 2) + row * (C * 2);
      const half8 pv = *(const half8*)(ob + (((2 * k8) ^ (row & 14)) << 3));
      half8 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        o[e] = (row & 1) ? pv[4 + e] : pv[e];
        o[4 + e] = (row & 1) ? pv[e] : pv[4 + e];
      }
      // streaming store: the block's output is read by the next launch, not this one
      __builtin_nontemporal_store(o, (half8*)(dst + (size_t)(yy * a.w + xx) * C + 8 * k8));
    }
  }
}

// ------------------------------------------------- pointwise, 256-row passes
// Contractions with 256-row passes and a plain or pixel-shuffled NHWC result
// (the patch embed, K = 192 frame values, and the 2C -> C fuse, K = 512, one
// pass each; the upsample, K = C, four passes = the four sub-positions of the
// shuffle): out^T[256 rows of the pass][128 pixels] = W act^T + b for one tile
// of 128 consecutive pixels per workgroup of 8 waves, the passes of a tile
// next to each other on one XCD (they share the tile's activations in L2).  Waves 0 .. 3 (one per SIMD) compute: wave w owns rows
// 64 w .. + 63 (two 32-row tiles) for all 128 pixels (four 32-pixel groups),
// so each weight fragment it holds feeds four MFMAs; the fragments come
// straight from global memory (L2) into registers as MFMA A operands, a few
// k-steps ahead.  Waves 4 .. 7 load: the activation tile (K / 64 slices of 128
// pixels x 64 contraction indices, 128-byte rows, 16-byte unit v of pixel p at
// position v ^ ((p / 2) & 7)) arrives by their direct global->LDS loads, at
// most DEPTH slices in flight, and each slice is released to the compute waves
// by a barrier once it is in (with every CU requesting its whole tile at once,
// the first slice would arrive only with the last).  Loads complete in order per wave,
// so keeping the activation loads (HBM) and the weight loads (L2) in different
// waves lets the weights stream while the activations are still arriving.  The
// sums (bias first, fp32) are rounded to fp16 once, parked in LDS and stored as
// 16-byte vectors (one contiguous block of 128 x 256 channels, or 512 bytes per
// output pixel of the shuffle).
template <int LOADER, int K, int EPI>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2))) void k_pw256_f16(PwArgs a) {
  constexpr int NK = K / 64;   // activation slices
  constexpr int NS = K / 16;   // MFMA k-steps
  constexpr int SLICE = 128 * 128;
  constexpr int PA = 3, PB = 2;  // prefetch distances (steps) of the A and B windows
  constexpr int DEPTH = 4;       // activation slices in flight
  constexpr int SMEM = NK * SLICE > 128 * 512 ? NK * SLICE : 128 * 512;
  static_assert(K % 64 == 0 && NK >= 2, "K is a multiple of 64, at least 128");
  __shared__ __attribute__((aligned(1024))) char smem[SMEM];
  static_assert(EPI == EP_NHWC || EPI == EP_UP || EPI == EP_REC, "plain or shuffled NHWC result, or the frame");
  // EP_REC: N = 192 rows in one pass; the weight image and the bias are
  // padded to 256 rows with zeros (wave 3's rows are computed and not stored)
  const int ntile = (a.P + 127) / 128, npass = (a.N + 255) / 256;
  const int lin = xcd_tile(blockIdx.x, gridDim.x);
  const int tile = lin / npass;
  if (tile >= ntile) return;
  const int n0 = (lin - tile * npass) * 256;  // first row of the pass
  // the upsample that follows the prior in an encode: workgroup 0 first adds
  // up the frame's rate partials
  if constexpr (EPI == EP_UP)
    if (a.bits_out && blockIdx.x == 0) block_sum_to(a.sum_base, a.n_sum, a.bits_out);
  const int lane = threadIdx.x & 63, h = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int myrow = lane & 31;

  floatx16 acc[2][4];  // (row tile c, pixel group g)
  if (wave >= 4) {
    // ---- loaders: slice kc is 16 direct loads, instruction i = (wave - 4) + 4 m
    const int lw = wave - 4;
    auto load_slice = [&](int kc) __attribute__((always_inline)) {
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        const int i = lw + 4 * m;
        const int S = i * 64 + lane;
        const int p = S >> 3, v = (S & 7) ^ ((p >> 1) & 7);
        const int gp = min(tile * 128 + p, a.P - 1);  // pixels past the end reload the last one
        dma16(pw_act_src<LOADER>(a, gp, kc, v, n0), smem + kc * SLICE + i * 1024);
      }
    };
#pragma unroll
    for (int kc = 0; kc < DEPTH && kc < NK; ++kc) load_slice(kc);
    auto release = [&](auto kcc) __attribute__((always_inline)) {
      constexpr int kc = decltype(kcc)::value;
      constexpr int later = (kc + DEPTH < NK ? kc + DEPTH : NK) - 1 - kc;  // slices requested after kc
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(4 * later) : "memory");  // slice kc is in
      lds_barrier();
      if constexpr (kc + DEPTH < NK) load_slice(kc + DEPTH);
    };
    unrolled_steps(release, std::make_integer_sequence<int, NK>{});
  } else {
    // ---- compute: rows 64 w + 32 c .., the accumulators start at the bias
    const half8* wf = (const half8*)a.wfrag + lane;  // fragment (row tile mt, k-step s) at [(mt NS + s) 64]
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const float* b = (const float*)a.bias + n0 + 64 * wave + 32 * c + 4 * h;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const floatx4 bv = *(const floatx4*)(b + 8 * q);
#pragma unroll
        for (int g = 0; g < 4; ++g)
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[c][g][4 * q + e] = bv[e];
      }
    }
    auto afrag = [&](int s, int c) __attribute__((always_inline)) {
      return wf[((size_t)(n0 / 32 + 2 * wave + c) * NS + s) * 64];
    };
    // B fragment of k-step s, group g: pixel 32 g + lane % 32, unit 2 (s % 4) + lane / 32 of slice s / 4
    auto bfrag = [&](int s, int g) __attribute__((always_inline)) {
      const int p = 32 * g + myrow, v = 2 * (s & 3) + h;
      return *(const half8*)(smem + (s >> 2) * SLICE + p * 128 + ((v ^ ((p >> 1) & 7)) << 4));
    };
    half8 qa[PA][2], qb[PB][4];
#pragma unroll
    for (int s = 0; s < PA; ++s)
#pragma unroll
      for (int c = 0; c < 2; ++c) qa[s][c] = afrag(s, c);
    lds_barrier();  // slice 0
#pragma unroll
    for (int s = 0; s < PB; ++s)
#pragma unroll
      for (int g = 0; g < 4; ++g) qb[s][g] = bfrag(s, g);
    // the barrier releasing slice kc + 1 is taken PB steps before slice kc
    // ends, so the B window runs across the slices
    auto step = [&](auto sc) __attribute__((always_inline)) {
      constexpr int s = decltype(sc)::value;
      if constexpr (s % 4 == 4 - PB && s / 4 + 1 < NK) lds_barrier();
      half8 A[2], B[4];
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        A[c] = qa[s % PA][c];
        if (s + PA < NS) qa[s % PA][c] = afrag(s + PA, c);
      }
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        B[g] = qb[s % PB][g];
        if (s + PB < NS) qb[s % PB][g] = bfrag(s + PB, g);
      }
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int g = 0; g < 4; ++g) acc[c][g] = mfma_f16(A[c], B[g], acc[c][g]);
      __builtin_amdgcn_sched_barrier(0);
    };
    static_assert(PB <= 4, "the slice barrier precedes the B reads of the next slice");
    unrolled_steps(step, std::make_integer_sequence<int, NS>{});
  }
  lds_barrier();  // every compute wave is done reading the slices
  // park: one rounding to fp16, row = tile pixel (512 bytes), 8-byte unit u of
  // the row at u ^ (row & 15)
  if (wave < 4) {
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int p = 32 * g + myrow;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int cc = 64 * wave + 32 * c + 8 * q + 4 * h;
          half4 o;
#pragma unroll
          for (int e = 0; e < 4; ++e) o[e] = (f16)acc[c][g][4 * q + e];
          *(half4*)(smem + p * 512 + (((cc >> 2) ^ (p & 15)) << 3)) = o;
        }
      }
  }
  lds_barrier();
  if constexpr (EPI == EP_REC) {
    // rows 64 c + 8 i + j: a 16-byte store covers the 8 frame pixels j of
    // (colour c, row i) of one 1/8-scale pixel; consecutive threads walk the
    // pixels, clamped to [0, 1] (the same as clamping before the rounding)
#pragma unroll
    for (int it = 0; it < 128 * 24 / 512; ++it) {
      const int idx = it * 512 + threadIdx.x;
      const int nl8 = idx >> 7, px = idx & 127;
      const int gp = tile * 128 + px;
      if (gp < a.P) {
        const half8 pv = *(const half8*)(smem + px * 512 + (((2 * nl8) ^ (px & 14)) << 3));
        const int c = nl8 >> 3, i = nl8 & 7;
        const int py = gp / a.w8, pxx = gp - py * a.w8;
        half8 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const f16 v0 = (px & 1) ? pv[4 + e] : pv[e], v1 = (px & 1) ? pv[e] : pv[4 + e];
          o[e] = __builtin_fminf16(__builtin_fmaxf16(v0, (f16)0.f), (f16)1.f);
          o[4 + e] = __builtin_fminf16(__builtin_fmaxf16(v1, (f16)0.f), (f16)1.f);
        }
        __builtin_nontemporal_store(o, (half8*)((f16*)a.dst + (size_t)c * a.H * a.W + (size_t)(8 * py + i) * a.W + 8 * pxx));
      }
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < 128 * 32 / 512; ++i) {
    const int idx = i * 512 + threadIdx.x;
    const int px = idx >> 5, k8 = idx & 31;  // tile pixel, 8-channel unit
    const int gp = tile * 128 + px;
    if (gp < a.P) {
      const char* ob = smem + px * 512;
      // units 2 k8 and 2 k8 + 1 are the aligned pair at 2 k8 ^ (px & 14), swapped when px is odd
      const half8 pv = *(const half8*)(ob + (((2 * k8) ^ (px & 14)) << 3));
      half8 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        o[e] = (px & 1) ? pv[4 + e] : pv[e];
        o[4 + e] = (px & 1) ? pv[e] : pv[4 + e];
      }
      size_t off;
      if constexpr (EPI == EP_NHWC) {
        off = (size_t)gp * a.Cdst + n0 + 8 * k8;
      } else {  // rows n = sp C + c: channel c of sub-position sp of the 2 x 2 shuffle
        const int C = a.Cdst, n = n0 + 8 * k8;
        const int sp = n / C, c = n - sp * C;
        const int w16 = a.w8 >> 1;
        const int Y = gp / w16, X = gp - Y * w16;
        off = (size_t)((2 * Y + (sp >> 1)) * a.w8 + 2 * X + (sp & 1)) * C + c;
      }
      *(half8*)((f16*)a.dst + off) = o;
    }
  }
}

template <int NT>
static hipError_t pw_dispatch(int loader, int epi, const PwArgs& a, hipStream_t st) {
  dim3 grid(grid_tiles(a.P) * (a.N / NT)), block(512);
#define NC_PW(L, E)                                                            \
  if (loader == L && epi == E) {                                               \
    launch(k_pw_f16<NT, L, E>, grid, block, st, a);                            \
    return hipGetLastError();                                                  \
  }
  NC_PW(LD_NHWC, EP_NHWC)
  NC_PW(LD_FRAME, EP_NHWC)
  NC_PW(LD_FRAME_CTX, EP_NHWC)
  if constexpr (NT != 256) {
    NC_PW(LD_DOWN, EP_NHWC)
    NC_PW(LD_NHWC, EP_UP)
    NC_PW(LD_UP_CTX, EP_UP)
    NC_PW(LD_NHWC, EP_REC)
    NC_PW(LD_NHWC, EP_LRELU)
    NC_PW(LD_NHWC, EP_RESID)
    NC_PW(LD_NHWC, EP_GATE)
  }
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
hipError_t launch_pw_f16(int loader, int epi, const PwArgs& a, hipStream_t st) {
  if (a.K % 64 || a.N % 64) return hipErrorInvalidValue;
  // The patch embed and the 2C -> C fuse have the widest activation tiles (K =
  // 192 frame values or 2C channels) at 1/8 scale (one tile per CU or more):
  // all N rows in one pass (N = 256: 48 KiB stages, one workgroup per CU) or
  // 128 rows per pass, so each tile is staged once or twice.  The 1/16-scale
  // kernels have 4x fewer tiles and keep 64-row passes to fill the CUs.
  if ((epi == EP_NHWC && a.N == 256 && a.Cdst == 256 &&
       ((loader == LD_FRAME && a.K == 192) || (loader == LD_NHWC && a.K == 512) ||
        (loader == LD_FRAME_CTX && a.K == 448))) ||
      (epi == EP_UP && a.N % 256 == 0 &&
       ((loader == LD_NHWC && a.K == 256) || (loader == LD_UP_CTX && a.K == 512 && a.Cdst == 256))) ||
      (epi == EP_REC && loader == LD_NHWC && a.K == 256 && a.N == 192 && a.C0 == 256 && a.ld0 == 0)) {
    dim3 grid(grid_tiles(a.P) * ((a.N + 255) / 256)), block(512);
    if (epi == EP_REC) launch(k_pw256_f16<LD_NHWC, 256, EP_REC>, grid, block, st, a);
    else if (epi == EP_UP && loader == LD_UP_CTX) launch(k_pw256_f16<LD_UP_CTX, 512, EP_UP>, grid, block, st, a);
    else if (epi == EP_UP) launch(k_pw256_f16<LD_NHWC, 256, EP_UP>, grid, block, st, a);
    else if (loader == LD_FRAME) launch(k_pw256_f16<LD_FRAME, 192, EP_NHWC>, grid, block, st, a);
    else if (loader == LD_FRAME_CTX) launch(k_pw256_f16<LD_FRAME_CTX, 448, EP_NHWC>, grid, block, st, a);
    else launch(k_pw256_f16<LD_NHWC, 512, EP_NHWC>, grid, block, st, a);
    return hipGetLastError();
  }
  if (epi == EP_NHWC && (loader == LD_FRAME || loader == LD_FRAME_CTX || (loader == LD_NHWC && a.K >= 512))) {
    if (a.N == 256) return pw_dispatch<256>(loader, epi, a, st);
    if (a.N % 128 == 0) return pw_dispatch<128>(loader, epi, a, st);
  }
  // the two halves of a wide DC block (C > 256) at 1/8 scale: 128-row passes
  if ((epi == EP_LRELU || epi == EP_RESID || epi == EP_GATE) && a.N % 128 == 0)
    return pw_dispatch<128>(loader, epi, a, st);
  return pw_dispatch<64>(loader, epi, a, st);
}

hipError_t launch_dcblock_f16(int C, bool gated, const BlockArgs& a, hipStream_t st) {
  // C = 256: the 128-pixels-per-wave kernel
  if (C == 256) return launch_dcblock128_f16(gated, a, st);
  dim3 grid(dc_grid(a.h, a.w)), block(512);
  switch (C * 2 + (gated ? 1 : 0)) {
    case 128: launch(k_dcblock_f16<64, false>, grid, block, st, a); break;
    case 256: launch(k_dcblock_f16<128, false>, grid, block, st, a); break;
    case 512: launch(k_dcblock_f16<256, false>, grid, block, st, a); break;
    case 129: launch(k_dcblock_f16<64, true>, grid, block, st, a); break;
    case 257: launch(k_dcblock_f16<128, true>, grid, block, st, a); break;
    case 513: launch(k_dcblock_f16<256, true>, grid, block, st, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Channels per workgroup: 64 (mu and s rows, 128 accumulator registers), which
// gives C / 64 workgroups per pixel tile.
// Prior head, quantiser and bits (Fig. 4 "Q", Supp. B.2) as the epilogue of
// the pointwise kernel: the head's rows are packed in passes of 32 mu rows
// followed by the 32 s rows of the same channels, so one workgroup holds both
// for its 128 latent pixels x 32 channels.  Bit partial sums: one per
// (tile, pass), reduced in a fixed order by k_reduce.
int prior_partials_f16(int C, int P) { return ((P + 127) / 128) * (C / 32); }

hipError_t launch_prior_f16(const PriorArgs& pa, hipStream_t st, int* n_partials) {
  if (pa.C % 32) return hipErrorInvalidValue;
  PwArgs a;
  std::memset(&a, 0, sizeof(a));
  a.wfrag = pa.wfrag;
  a.bias = pa.bias;
  a.K = pa.K ? pa.K : pa.C;
  a.N = pa.N ? pa.N : 2 * pa.C;
  a.ld0 = pa.ld0;
  a.c_off = pa.c_off;
  a.add = pa.add;
  a.add_ld = pa.add_ld;
  a.add_s = pa.add_s;
  a.add_c0 = pa.add_c0;
  a.add_f32 = pa.add_f32;
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
  a.k_out = pa.k_out;
  a.scales = pa.scales;
  if (n_partials) *n_partials = ((pa.P + 127) / 128) * (a.N / 64);
  return pw_dispatch<64>(LD_NHWC, pa.decode == 2 ? EP_SCALES : pa.decode ? EP_PRIOR_DEC : EP_PRIOR, a, st);
}

hipError_t launch_zquant_f16(const PwArgs& a, hipStream_t st, int* n_partials) {
  if (a.N != 64 || a.K % 64) return hipErrorInvalidValue;
  if (n_partials) *n_partials = (a.P + 127) / 128;
  return pw_dispatch<64>(LD_DOWN, EP_ZQUANT, a, st);
}

}  // namespace nc
