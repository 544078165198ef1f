// Small kernels: deterministic bit reduction, the standalone rate estimate,
// zero fill, and state layout conversion (channels-last <-> planar).
#include "common.hpp"
#include "internal.hpp"

namespace nc {

// One workgroup; thread t sums partials t, t+256, ... in order, then a fixed
// LDS tree.  The result does not depend on timing.
__global__ __launch_bounds__(256) void k_reduce(const double* part, int n, double* out) {
  __shared__ double sh[256];
  double v = 0.0;
  for (int i = threadIdx.x; i < n; i += 256) v += part[i];
  sh[threadIdx.x] = v;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if ((int)threadIdx.x < s) sh[threadIdx.x] += sh[threadIdx.x + s];
    __syncthreads();
  }
  if (threadIdx.x == 0) *out = sh[0];
}

// Block b owns elements [b*chunk, min(n, (b+1)*chunk)); chunk depends only on n.
// The scale of element i is sigma[i] (float32), or on the integer path
// sigma_tab[s[i] + 32768] for the prior's int16 scale output s (a table of
// max(softplus(s / 512), 0.11) over every int16 value).
template <bool INT_SCALE>
__global__ __launch_bounds__(256) void k_bits(const int16_t* q, const void* scale, const float* sigma_tab, int64_t n,
                                              int64_t chunk, double* part) {
  const int64_t lo = (int64_t)blockIdx.x * chunk;
  const int64_t hi = min(n, lo + chunk);
  double v = 0.0;
  for (int64_t i = lo + threadIdx.x; i < hi; i += 256) {
    float sg;
    if constexpr (INT_SCALE) sg = sigma_tab[(int)((const int16_t*)scale)[i] + 32768];
    else sg = ((const float*)scale)[i];
    v += (double)symbol_bits((float)q[i], sg);
  }
  __shared__ double red[4];
  v = wave_sum(v);
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[wave] = v;
  __syncthreads();
  if (threadIdx.x == 0) part[blockIdx.x] = ((red[0] + red[1]) + red[2]) + red[3];
}

__global__ void k_fill_zero(uint32_t* p, size_t n) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) p[i] = 0u;
}

// planar[c*P + p] = nhwc[p*C + c] (2-byte elements)
__global__ void k_nhwc_to_planar(const uint16_t* src, uint16_t* dst, int C, int P) {
  const size_t n = (size_t)C * P;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    const size_t c = i / P, p = i - c * P;
    dst[i] = src[p * C + c];
  }
}

__global__ void k_planar_to_nhwc(const uint16_t* src, uint16_t* dst, int C, int P) {
  const size_t n = (size_t)C * P;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    const size_t p = i / C, c = i - p * C;
    dst[i] = src[c * P + p];
  }
}

// One workgroup per (64-pixel, 32-channel) tile: the planar symbols of the
// tile are staged through LDS (coalesced row reads), then each thread forms
// 8 consecutive channels of one pixel and stores them as one 16-byte vector.
// Channels c < C of q (planar, C x P) go to channel c_off + c of mu and yhat
// (NHWC, row stride ld); a NULL mu is zero.
template <bool IS_INT>
__global__ __launch_bounds__(256) void k_yhat_from_q(const int16_t* q, const void* mu, void* yhat, int C, int P, int ld,
                                                     int c_off) {
  __shared__ int16_t qs[32][64 + 2];
  const int ntp = (P + 63) / 64;
  const int tp = blockIdx.x % ntp, tc = blockIdx.x / ntp;
  const int p0 = tp * 64, c0 = tc * 32;
  for (int i = threadIdx.x; i < 32 * 64; i += 256) {
    const int cc = i >> 6, pp = i & 63;
    qs[cc][pp] = p0 + pp < P ? q[(size_t)(c0 + cc) * P + p0 + pp] : (int16_t)0;
  }
  __syncthreads();
  const int pp = threadIdx.x >> 2, g8 = threadIdx.x & 3;
  const int gp = p0 + pp;
  if (gp >= P) return;
  const size_t off = (size_t)gp * ld + c_off + c0 + 8 * g8;
  if constexpr (IS_INT) {
    shortx8 m = {};
    if (mu) m = *(const shortx8*)((const int16_t*)mu + off);
    shortx8 o;
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = (short)clip16(512 * (int)qs[8 * g8 + e][pp] + (int)m[e]);
    *(shortx8*)((int16_t*)yhat + off) = o;
  } else {
    floatx4 m0 = {}, m1 = {};
    if (mu) {
      m0 = *(const floatx4*)((const float*)mu + off);
      m1 = *(const floatx4*)((const float*)mu + off + 4);
    }
    half8 o;
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = (f16)((float)qs[8 * g8 + e][pp] + (e < 4 ? m0[e] : m1[e - 4]));
    *(half8*)((f16*)yhat + off) = o;
  }
}

hipError_t launch_yhat_from_q(const int16_t* q, const void* mu, void* yhat, int C, int P, bool is_int,
                              hipStream_t st, int ld, int c_off) {
  if (C % 32 || c_off % 8) return hipErrorInvalidValue;
  if (!ld) ld = C;
  const dim3 grid(((P + 63) / 64) * (C / 32));
  if (is_int) launch(k_yhat_from_q<true>, grid, dim3(256), st, q, mu, yhat, C, P, ld, c_off);
  else launch(k_yhat_from_q<false>, grid, dim3(256), st, q, mu, yhat, C, P, ld, c_off);
  return hipGetLastError();
}

hipError_t launch_reduce(const double* partials, int n, double* out, hipStream_t st) {
  launch(k_reduce, dim3(1), dim3(256), st, partials, n, out);
  return hipGetLastError();
}

hipError_t launch_estimate_bits(const int16_t* q, const void* scale, const float* sigma_tab, int64_t n,
                                double* partials, double* out, hipStream_t st) {
  const int64_t chunk = n > 0 ? (n + kBitsBlocks - 1) / kBitsBlocks : 1;
  if (sigma_tab)
    launch(k_bits<true>, dim3(kBitsBlocks), dim3(256), st, q, scale, sigma_tab, n, chunk, partials);
  else
    launch(k_bits<false>, dim3(kBitsBlocks), dim3(256), st, q, scale, sigma_tab, n, chunk, partials);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_reduce(partials, kBitsBlocks, out, st);
}

hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t st) {
  const size_t n = bytes / 4;
  if (n == 0) return hipSuccess;
  const int blocks = (int)std::min<size_t>((n + 255) / 256, 4096);
  launch(k_fill_zero, dim3(blocks), dim3(256), st, (uint32_t*)p, n);
  return hipGetLastError();
}

hipError_t launch_nhwc_to_planar(const void* src, void* dst, int C, int P, hipStream_t st) {
  const size_t n = (size_t)C * P;
  const int blocks = (int)std::min<size_t>((n + 255) / 256, 8192);
  launch(k_nhwc_to_planar, dim3(blocks), dim3(256), st, (const uint16_t*)src, (uint16_t*)dst, C, P);
  return hipGetLastError();
}

hipError_t launch_planar_to_nhwc(const void* src, void* dst, int C, int P, hipStream_t st) {
  const size_t n = (size_t)C * P;
  const int blocks = (int)std::min<size_t>((n + 255) / 256, 8192);
  launch(k_planar_to_nhwc, dim3(blocks), dim3(256), st, (const uint16_t*)src, (uint16_t*)dst, C, P);
  return hipGetLastError();
}

}  // namespace nc
