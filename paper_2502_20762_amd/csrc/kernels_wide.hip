// Depthwise 3x3 of a DC block as a kernel of its own, for the wide blocks
// (C > 256: the Large model's width, Supp. "Performance for a Large Model")
// whose weights and hidden layer do not fit the LDS of one CU in a fused
// block.  A wide block is three launches: this kernel, the pointwise C -> 2C
// with the LeakyReLU epilogue, the pointwise 2C -> C with the residual
// epilogue (Supp. B.1; Alg. 1 on the integer path).
//
// One thread per (pixel, 8 channels): consecutive threads take consecutive
// channel groups of a pixel, so every tap is a coalesced 16-byte load of the
// NHWC map (the 3 x 3 neighbourhood is re-read from L2 by the neighbours);
// the thread's 9 x 8 weights and 8 biases are shared by all pixels and stay
// in L1 / L2.
#include "common.hpp"
#include "internal.hpp"

namespace nc {

// fp16: a = b + sum over (ky, kx) of w * z in fp32 (taps row by row, the
// order of the fused block), one rounding to fp16; taps outside the map are
// zero and skipped (fma with 0 leaves the sum unchanged).
__global__ __launch_bounds__(256) void k_dw3x3_f16(const f16* z, const uint32_t* dww, f16* out, int C, int h, int w) {
  const int G = C / 8;
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= (int64_t)h * w * G) return;
  const int g = (int)(t % G);
  const int p = (int)(t / G);
  const int y = p / w, x = p - y * w;
  // 4 channel pairs: 12 words each (9 taps as fp16 pairs, 2 fp32 biases, pad)
  half2 wt[4][9];
  float acc[8];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t* q = dww + 12 * (4 * g + i);
    const intx4 q0 = *(const intx4*)q, q1 = *(const intx4*)(q + 4), q2 = *(const intx4*)(q + 8);
    // each word is copied to a scalar before the bit cast (a bit cast of the
    // vector element itself was compiled as a cast of element 0)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int x0 = q0[e], x1 = q1[e];
      wt[i][e] = __builtin_bit_cast(half2, x0);
      wt[i][4 + e] = __builtin_bit_cast(half2, x1);
    }
    const int x8 = q2[0], xb0 = q2[1], xb1 = q2[2];
    wt[i][8] = __builtin_bit_cast(half2, x8);
    acc[2 * i] = __builtin_bit_cast(float, xb0);
    acc[2 * i + 1] = __builtin_bit_cast(float, xb1);
  }
#pragma unroll
  for (int ky = 0; ky < 3; ++ky) {
    const int yy = y + ky - 1;
    if (yy < 0 || yy >= h) continue;
#pragma unroll
    for (int kx = 0; kx < 3; ++kx) {
      const int xx = x + kx - 1;
      if (xx < 0 || xx >= w) continue;
      const half8 v = *(const half8*)(z + ((size_t)yy * w + xx) * C + 8 * g);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const half2 ww = wt[i][3 * ky + kx];
        acc[2 * i] = fmaf((float)ww[0], (float)v[2 * i], acc[2 * i]);
        acc[2 * i + 1] = fmaf((float)ww[1], (float)v[2 * i + 1], acc[2 * i + 1]);
      }
    }
  }
  half8 o;
#pragma unroll
  for (int e = 0; e < 8; ++e) o[e] = (f16)acc[e];
  *(half8*)(out + (size_t)p * C + 8 * g) = o;
}

// int16: a_i = clip(RHE((512 b + sum w_i z_i) / 8192)) in wrapping int32
// (Alg. 1; the sum is the same in any order).
__global__ __launch_bounds__(256) void k_dw3x3_i16(const int16_t* z, const uint32_t* dww, int16_t* out, int C, int h,
                                                   int w) {
  const int G = C / 8;
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= (int64_t)h * w * G) return;
  const int g = (int)(t % G);
  const int p = (int)(t / G);
  const int y = p / w, x = p - y * w;
  // 2 channel quads: 24 words each (per tap the int16 pairs (c, c+1), (c+2,
  // c+3); then the 4 biases 512 b; 2 pad words)
  uint32_t wq[2][18];
  int acc[8];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const uint32_t* q = dww + 24 * (2 * g + i);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const intx4 v = *(const intx4*)(q + 4 * u);
#pragma unroll
      for (int e = 0; e < 4; ++e) wq[i][4 * u + e] = (uint32_t)v[e];
    }
    const intx4 v4 = *(const intx4*)(q + 16);
    wq[i][16] = (uint32_t)v4[0];
    wq[i][17] = (uint32_t)v4[1];
    acc[4 * i] = v4[2];
    acc[4 * i + 1] = v4[3];
    const intx4 v5 = *(const intx4*)(q + 20);
    acc[4 * i + 2] = v5[0];
    acc[4 * i + 3] = v5[1];
  }
#pragma unroll
  for (int ky = 0; ky < 3; ++ky) {
    const int yy = y + ky - 1;
    if (yy < 0 || yy >= h) continue;
#pragma unroll
    for (int kx = 0; kx < 3; ++kx) {
      const int xx = x + kx - 1;
      if (xx < 0 || xx >= w) continue;
      const shortx8 v = *(const shortx8*)(z + ((size_t)yy * w + xx) * C + 8 * g);
      const int tap = 3 * ky + kx;
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          const uint32_t pr = wq[i][2 * tap + e];
          const int c = 4 * i + 2 * e;
          acc[c] = (int)((uint32_t)acc[c] + (uint32_t)((int)(short)(pr & 0xFFFFu) * (int)v[c]));
          acc[c + 1] = (int)((uint32_t)acc[c + 1] + (uint32_t)((int)(short)(pr >> 16) * (int)v[c + 1]));
        }
    }
  }
  shortx8 o;
#pragma unroll
  for (int e = 0; e < 8; ++e) o[e] = (short)rescale13(acc[e]);
  *(shortx8*)(out + (size_t)p * C + 8 * g) = o;
}

namespace {
dim3 dw_grid(int C, int h, int w) { return dim3((unsigned)(((int64_t)h * w * (C / 8) + 255) / 256)); }
}  // namespace

hipError_t launch_dw3x3_f16(const void* src, const void* dww, void* dst, int C, int h, int w, hipStream_t st) {
  if (C % 8 || h <= 0 || w <= 0) return hipErrorInvalidValue;
  launch(k_dw3x3_f16, dw_grid(C, h, w), dim3(256), st, (const f16*)src, (const uint32_t*)dww, (f16*)dst, C, h, w);
  return hipGetLastError();
}

hipError_t launch_dw3x3_i16(const void* src, const void* dww, void* dst, int C, int h, int w, hipStream_t st) {
  if (C % 8 || h <= 0 || w <= 0) return hipErrorInvalidValue;
  launch(k_dw3x3_i16, dw_grid(C, h, w), dim3(256), st, (const int16_t*)src, (const uint32_t*)dww, (int16_t*)dst, C,
         h, w);
  return hipGetLastError();
}

}  // namespace nc
