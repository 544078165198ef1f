// fp16 path kernels (fp16 storage, fp32 MFMA accumulation) for gfx950.
//
// k_pw_f16      pointwise / patch-embed / 2x2-s2 / upsample / reconstruction
//               contractions (out^T = W * act^T + b) with gather-on-load and
//               scatter-on-store, one wave = 32 pixels x NT output channels.
// k_dcblock_f16 one whole DC block (Supp. B.1): depthwise 3x3 computed into
//               registers, pw C->2C + LeakyReLU chained into pw 2C->C through
//               registers 32 hidden channels at a time, residual add.
// k_prior_f16   1x1 prior head on yhat_{t-1}, quantiser, yhat_t and the
//               per-tile bit partial sums (Fig. 4 "Q", Supp. B.2).
#include "common.hpp"
#include "internal.hpp"

namespace nc {

template <int LOADER>
__device__ __forceinline__ half8 load_b_f16(const PwArgs& a, int p, int k0) {
  if constexpr (LOADER == LD_NHWC) {
    if (k0 < a.C0) return *(const half8*)((const f16*)a.src0 + (size_t)p * a.C0 + k0);
    return *(const half8*)((const f16*)a.src1 + (size_t)p * a.C1 + (k0 - a.C0));
  } else if constexpr (LOADER == LD_FRAME) {
    const int py = p / a.w8, px = p - py * a.w8;
    const int c = k0 >> 6, i = (k0 >> 3) & 7;
    return *(const half8*)((const f16*)a.src0 + (size_t)c * a.H * a.W + (size_t)(8 * py + i) * a.W + 8 * px);
  } else {
    const int w16 = a.w8 >> 1;
    const int Y = p / w16, X = p - Y * w16;
    const int tap = k0 / a.Csrc, c = k0 - tap * a.Csrc;
    const int pix = (2 * Y + (tap >> 1)) * a.w8 + 2 * X + (tap & 1);
    return *(const half8*)((const f16*)a.src0 + (size_t)pix * a.Csrc + c);
  }
}

template <int NT, int LOADER, int EPI>
__global__ __launch_bounds__(256) void k_pw_f16(PwArgs a) {
  constexpr int MT = NT / 32;
  const int ntile = (a.P + 127) / 128;
  const int tile = xcd_tile(blockIdx.x, gridDim.x);
  if (tile >= ntile) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, h = lane >> 5;
  const int p = tile * 128 + wave * 32 + (lane & 31);
  const bool valid = p < a.P;
  const int mt0 = blockIdx.y * MT;
  const int ks = a.K / 16;
  const half8* wf = (const half8*)a.wfrag;

  floatx16 acc[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) acc[t] = floatx16{};

  for (int s = 0; s < ks; ++s) {
    half8 b = {};
    if (valid) b = load_b_f16<LOADER>(a, p, 16 * s + 8 * h);
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      const half8 w = wf[((size_t)(mt0 + t) * ks + s) * 64 + lane];
      acc[t] = mfma_f16(w, b, acc[t]);
    }
  }
  if (!valid) return;

  const float* bias = (const float*)a.bias;
#pragma unroll
  for (int t = 0; t < MT; ++t) {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int n = 32 * (mt0 + t) + 8 * g + 4 * h;
      const floatx4 bv = *(const floatx4*)(bias + n);
      half4 o;
      if constexpr (EPI == EP_REC) {
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = (f16)fminf(fmaxf(acc[t][4 * g + e] + bv[e], 0.f), 1.f);
        const int c = n >> 6, i = (n >> 3) & 7, j0 = n & 7;
        const int py = p / a.w8, px = p - py * a.w8;
        *(half4*)((f16*)a.dst + (size_t)c * a.H * a.W + (size_t)(8 * py + i) * a.W + 8 * px + j0) = o;
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = (f16)(acc[t][4 * g + e] + bv[e]);
        if constexpr (EPI == EP_NHWC) {
          *(half4*)((f16*)a.dst + (size_t)p * a.Cdst + n) = o;
        } else {  // EP_UP: row n = sp * C + c
          const int C = a.Cdst;
          const int sp = n / C, c = n - sp * C;
          const int w16 = a.w8 >> 1;
          const int Y = p / w16, X = p - Y * w16;
          const int pix = (2 * Y + (sp >> 1)) * a.w8 + 2 * X + (sp & 1);
          *(half4*)((f16*)a.dst + (size_t)pix * C + c) = o;
        }
      }
    }
  }
}

template <int C>
__global__ __launch_bounds__(256) void k_dcblock_f16(BlockArgs a) {
  constexpr int KS = C / 16;       // k-steps over the C input channels
  constexpr int NCH = 2 * C / 32;  // hidden chunks of 32
  constexpr int MT = C / 32;       // output row tiles
  constexpr int KS2 = 2 * C / 16;  // k-steps over the hidden channels
  const int P = a.h * a.w;
  const int ntile = (P + 127) / 128;
  const int tile = xcd_tile(blockIdx.x, gridDim.x);
  if (tile >= ntile) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, h = lane >> 5;
  const int p = tile * 128 + wave * 32 + (lane & 31);
  const bool valid = p < P;
  const int y = valid ? p / a.w : 0, x = valid ? p - y * a.w : 0;
  const f16* z = (const f16*)a.src;

  // depthwise 3x3 (+ bias) for this lane's pixel, channels 16s + 8h + e.
  half8 av[KS];
  {
    const half8* dww = (const half8*)a.dww;
    const float* dwb = (const float*)a.dwb;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int c0 = 16 * s + 8 * h;
      float acc[8];
      const floatx4 b0 = *(const floatx4*)(dwb + c0), b1v = *(const floatx4*)(dwb + c0 + 4);
#pragma unroll
      for (int e = 0; e < 4; ++e) { acc[e] = b0[e]; acc[4 + e] = b1v[e]; }
#pragma unroll
      for (int ky = 0; ky < 3; ++ky) {
        const int yy = y + ky - 1;
#pragma unroll
        for (int kx = 0; kx < 3; ++kx) {
          const int xx = x + kx - 1;
          if (valid && yy >= 0 && yy < a.h && xx >= 0 && xx < a.w) {
            const half8 v = *(const half8*)(z + (size_t)(yy * a.w + xx) * C + c0);
            const half8 wv = dww[(ky * 3 + kx) * (C / 8) + (c0 >> 3)];
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[e] = fmaf((float)wv[e], (float)v[e], acc[e]);
          }
        }
      }
      half8 o;
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = valid ? (f16)acc[e] : (f16)0.f;
      av[s] = o;
    }
  }

  const half8* w1 = (const half8*)a.w1;
  const half8* w2 = (const half8*)a.w2;
  const float* b1 = (const float*)a.b1;
  floatx16 out[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) out[t] = floatx16{};

  for (int j = 0; j < NCH; ++j) {
    floatx16 hacc = {};
#pragma unroll
    for (int s = 0; s < KS; ++s) hacc = mfma_f16(w1[((size_t)j * KS + s) * 64 + lane], av[s], hacc);
    half8 g0, g1;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const floatx4 bv = *(const floatx4*)(b1 + 32 * j + 8 * g + 4 * h);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const f16 v = (f16)leaky(hacc[4 * g + e] + bv[e]);
        if (g < 2) g0[4 * g + e] = v; else g1[4 * (g - 2) + e] = v;
      }
    }
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      out[t] = mfma_f16(w2[((size_t)t * KS2 + 2 * j) * 64 + lane], g0, out[t]);
      out[t] = mfma_f16(w2[((size_t)t * KS2 + 2 * j + 1) * 64 + lane], g1, out[t]);
    }
  }
  if (!valid) return;

  const float* b2 = (const float*)a.b2;
  f16* dst = (f16*)a.dst;
#pragma unroll
  for (int t = 0; t < MT; ++t) {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int c = 32 * t + 8 * g + 4 * h;
      const floatx4 bv = *(const floatx4*)(b2 + c);
      const half4 zv = *(const half4*)(z + (size_t)p * C + c);
      half4 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = (f16)(out[t][4 * g + e] + bv[e] + (float)zv[e]);
      *(half4*)(dst + (size_t)p * C + c) = o;
    }
  }
}

// Prior head, quantiser and bits.  One wave = 32 latent pixels x CH channels
// (their mu rows and their s rows).  Workgroup partial sums are written per
// (tile, channel slice) and reduced in a fixed order by k_reduce.
template <int CH, bool DECODE>
__global__ __launch_bounds__(256) void k_prior_f16(PriorArgs a) {
  constexpr int MT = CH / 32;
  const int ntile = (a.P + 127) / 128;
  const int tile = xcd_tile(blockIdx.x, gridDim.x);
  if (tile >= ntile) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, h = lane >> 5;
  const int p = tile * 128 + wave * 32 + (lane & 31);
  const bool valid = p < a.P;
  const int C = a.C;
  const int ct0 = blockIdx.y * MT;
  const int ks = C / 16;
  const half8* wf = (const half8*)a.wfrag;
  const f16* yp = (const f16*)a.yhat_prev;

  floatx16 amu[MT], asg[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) { amu[t] = floatx16{}; asg[t] = floatx16{}; }
  for (int s = 0; s < ks; ++s) {
    half8 b = {};
    if (valid) b = *(const half8*)(yp + (size_t)p * C + 16 * s + 8 * h);
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      amu[t] = mfma_f16(wf[((size_t)(ct0 + t) * ks + s) * 64 + lane], b, amu[t]);
      if constexpr (!DECODE) asg[t] = mfma_f16(wf[((size_t)(C / 32 + ct0 + t) * ks + s) * 64 + lane], b, asg[t]);
    }
  }

  const float* bias = (const float*)a.bias;
  double bsum = 0.0;
  if (valid) {
#pragma unroll
    for (int t = 0; t < MT; ++t) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int c = 32 * (ct0 + t) + 8 * g + 4 * h;
        const floatx4 bm = *(const floatx4*)(bias + c);
        half4 yh;
        if constexpr (DECODE) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            // same operation order as the encoder: mu first, then q + mu
            const float mu = amu[t][4 * g + e] + bm[e];
            const float q = (float)a.q_in[(size_t)(c + e) * a.P + p];
            yh[e] = (f16)(q + mu);
          }
        } else {
          const floatx4 bs = *(const floatx4*)(bias + C + c);
          const half4 yv = *(const half4*)((const f16*)a.y + (size_t)p * C + c);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float mu = amu[t][4 * g + e] + bm[e];
            float q = rintf((float)yv[e] - mu);
            q = fminf(fmaxf(q, -32768.f), 32767.f);
            a.q_out[(size_t)(c + e) * a.P + p] = (int16_t)q;
            yh[e] = (f16)(q + mu);
            bsum += (double)symbol_bits(q, softplus_sigma(asg[t][4 * g + e] + bs[e]));
          }
        }
        *(half4*)((f16*)a.yhat_new + (size_t)p * C + c) = yh;
      }
    }
  }
  if constexpr (DECODE) return;
  __shared__ double red[4];
  bsum = wave_sum(bsum);
  if (lane == 0) red[wave] = bsum;
  __syncthreads();
  if (threadIdx.x == 0) a.partials[(size_t)tile * gridDim.y + blockIdx.y] = ((red[0] + red[1]) + red[2]) + red[3];
}

template <int NT>
static hipError_t pw_dispatch(int loader, int epi, const PwArgs& a, hipStream_t st) {
  dim3 grid(grid_tiles(a.P), a.N / NT), block(256);
#define NC_PW(L, E)                                                            \
  if (loader == L && epi == E) {                                               \
    hipLaunchKernelGGL((k_pw_f16<NT, L, E>), grid, block, 0, st, a);           \
    return hipGetLastError();                                                  \
  }
  NC_PW(LD_NHWC, EP_NHWC)
  NC_PW(LD_FRAME, EP_NHWC)
  NC_PW(LD_DOWN, EP_NHWC)
  NC_PW(LD_NHWC, EP_UP)
  NC_PW(LD_NHWC, EP_REC)
#undef NC_PW
  return hipErrorInvalidValue;
}

hipError_t launch_pw_f16(int loader, int epi, const PwArgs& a, hipStream_t st) {
  if (a.N % 256 == 0) return pw_dispatch<256>(loader, epi, a, st);
  if (a.N % 192 == 0) return pw_dispatch<192>(loader, epi, a, st);
  if (a.N % 128 == 0) return pw_dispatch<128>(loader, epi, a, st);
  if (a.N % 64 == 0) return pw_dispatch<64>(loader, epi, a, st);
  return hipErrorInvalidValue;
}

hipError_t launch_dcblock_f16(int C, const BlockArgs& a, hipStream_t st) {
  dim3 grid(grid_tiles(a.h * a.w)), block(256);
  switch (C) {
    case 64: hipLaunchKernelGGL((k_dcblock_f16<64>), grid, block, 0, st, a); break;
    case 128: hipLaunchKernelGGL((k_dcblock_f16<128>), grid, block, 0, st, a); break;
    case 256: hipLaunchKernelGGL((k_dcblock_f16<256>), grid, block, 0, st, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

int prior_partials_f16(int C, int P) { return grid_tiles(P) * (C >= 128 ? C / 128 : 1); }

hipError_t launch_prior_f16(const PriorArgs& a, hipStream_t st, int* n_partials) {
  const int ch = a.C >= 128 ? 128 : a.C;
  dim3 grid(grid_tiles(a.P), a.C / ch), block(256);
  if (n_partials) *n_partials = ((a.P + 127) / 128) * (a.C / ch);
  if (ch == 128 && a.decode) hipLaunchKernelGGL((k_prior_f16<128, true>), grid, block, 0, st, a);
  else if (ch == 128) hipLaunchKernelGGL((k_prior_f16<128, false>), grid, block, 0, st, a);
  else if (ch == 64 && a.decode) hipLaunchKernelGGL((k_prior_f16<64, true>), grid, block, 0, st, a);
  else if (ch == 64) hipLaunchKernelGGL((k_prior_f16<64, false>), grid, block, 0, st, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace nc
