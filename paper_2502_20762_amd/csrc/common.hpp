// Shared device helpers for the gfx950 kernels of ncodec.
//
// Every GEMM-shaped step is computed "transposed": out^T[rows = output
// channels][cols = pixels] = W[rows][K] * act^T[K][pixels].  The weights are
// the MFMA A operand (pre-packed in fragment order, one coalesced 1 KiB load
// per wave per fragment), the activations are the B operand (8 or 16
// consecutive channels of one pixel per lane, a 16/32-byte load from the
// channels-last feature map), and in the 32x32 accumulator layout each lane
// owns one pixel column, so chained contractions can feed one MFMA's result
// straight into the next as its B operand without a trip through LDS.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef _Float16 f16;
typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half4 __attribute__((ext_vector_type(4)));
typedef _Float16 half2 __attribute__((ext_vector_type(2)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef int intx4 __attribute__((ext_vector_type(4)));
typedef int intx3 __attribute__((ext_vector_type(3)));
typedef int intx2 __attribute__((ext_vector_type(2)));
typedef int intx16 __attribute__((ext_vector_type(16)));
typedef short shortx8 __attribute__((ext_vector_type(8)));
typedef short shortx4 __attribute__((ext_vector_type(4)));

namespace nc {

constexpr int kWave = 64;
constexpr int kWavesPerWG = 4;
constexpr int kPxPerWave = 32;
constexpr int kPxPerWG = kWave * kWavesPerWG / 2;  // 128 pixels per workgroup
constexpr int kNumXCD = 8;

// v_mfma_f32_32x32x16_f16: A lane l = row l%32, k 8*(l/32)+e; B lane l = k 8*(l/32)+e, col l%32.
__device__ __forceinline__ floatx16 mfma_f16(half8 a, half8 b, floatx16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}
// v_mfma_i32_32x32x32_i8: A lane l = row l%32, k 16*(l/32)+e (bytes); int32 accumulate wraps.
__device__ __forceinline__ intx16 mfma_i8(intx4 a, intx4 b, intx16 c) {
  return __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c, 0, 0, 0);
}

// Row of accumulator register r for lane half h in the 32x32 output layout.
__host__ __device__ constexpr int drow(int r, int h) { return 8 * (r / 4) + 4 * h + (r % 4); }

// Workgroup -> tile mapping that gives each XCD a contiguous range of tiles
// (workgroups are dispatched round-robin over the 8 XCDs), so neighbouring
// tiles that share halo rows hit the same L2.  The grid is a multiple of 8.
__device__ __forceinline__ int xcd_tile(int bid, int nblk) {
  const int per = nblk / kNumXCD;
  return (bid % kNumXCD) * per + bid / kNumXCD;
}

// round-half-to-even of a / 2^s (1 <= s <= 30), from floor and remainder.
__device__ __forceinline__ int rhe_shift(int a, int s) {
  const int fl = a >> s;                       // arithmetic shift = floor
  const int r = a & ((1 << s) - 1);            // a - fl * 2^s, in [0, 2^s)
  const int half = 1 << (s - 1);
  return fl + (int)((r > half) | ((r == half) & (fl & 1)));
}
__device__ __forceinline__ int clip16(int v) { return min(max(v, -32768), 32767); }

// Alg. 1's rescale of an int32 convolution sum, clip(RHE(a / 8192)), for any
// int32 a.  |a| >= 2^28 saturates either way, so a is first clamped to
// +-2^28; then the round-half-even bias can be added without overflow:
// RHE(a / 2^s) = (a + 2^(s-1) - 1 + ((a >> s) & 1)) >> s.
__device__ __forceinline__ int rescale13(int a) {
  const int ac = min(max(a, -(1 << 28)), 1 << 28);
  return clip16((ac + 4095 + ((ac >> 13) & 1)) >> 13);
}

// Combine the three partial products of an int16 x int16 contraction done as
// int8 digits (x = 256 xh + xl' + 128, w = 256 wh + wl) in wrapping int32.
__device__ __forceinline__ int combine_i16(int hh, int mid, int ll, int corr) {
  const uint32_t v = ((uint32_t)hh << 16) + ((uint32_t)mid << 8) + (uint32_t)ll + (uint32_t)corr;
  return (int)v;
}

// Split 4 int16 values (two dwords) into their high bytes (signed) and their
// low bytes offset by -128 (xl' = (x & 255) - 128, i.e. the low byte ^ 0x80).
__device__ __forceinline__ void split4(uint32_t d0, uint32_t d1, uint32_t& hi, uint32_t& lo) {
  hi = ((d0 >> 8) & 0xFFu) | ((d0 >> 24) << 8) | (((d1 >> 8) & 0xFFu) << 16) | ((d1 >> 24) << 24);
  lo = ((d0 & 0xFFu) | (((d0 >> 16) & 0xFFu) << 8) | ((d1 & 0xFFu) << 16) | (((d1 >> 16) & 0xFFu) << 24)) ^
       0x80808080u;
}

// Split 16 int16 values (8 dwords) into hi / lo int8 fragments.
__device__ __forceinline__ void split16(const uint32_t* d, intx4& hi, intx4& lo) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint32_t h, l;
    split4(d[2 * i], d[2 * i + 1], h, l);
    hi[i] = (int)h;
    lo[i] = (int)l;
  }
}

// Direct global->LDS load of 16 bytes per lane: lane l's bytes land at
// lds_wave_base + 16 l (the base is wave-uniform and goes through M0).  It is
// issued from inline asm so that the compiler does not treat every later LDS
// read as dependent on it (it would otherwise wait for all outstanding loads
// before each LDS read); callers wait explicitly with s_waitcnt vmcnt(N),
// counting these loads, before reading the destination.
__device__ __forceinline__ void dma16(const void* g, const void* lds_wave_base) {
  const uint32_t m = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)lds_wave_base;
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(m) : "memory", "m0");
}

// The same with a wave-uniform 64-bit base in SGPRs and a per-lane 32-bit
// byte offset (one VGPR shared by every such load of a kernel, instead of a
// 64-bit address per load).
__device__ __forceinline__ void dma16s(const void* sbase, uint32_t voff, const void* lds_wave_base) {
  const uint32_t m = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)lds_wave_base;
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(sbase), "s"(m)
               : "memory", "m0");
}

// Read-only kernel data seen through the constant address space: loads at
// wave-uniform addresses become scalar loads.
typedef const __attribute__((address_space(4))) float cfloat;
typedef const __attribute__((address_space(4))) int32_t cint;
typedef const __attribute__((address_space(4))) half8 chalf8;
typedef const __attribute__((address_space(4))) shortx8 cshortx8;
typedef const __attribute__((address_space(4))) intx4 cintx4;

// Workgroup barrier for LDS hand-offs inside a pipelined loop.  It waits for
// this wave's LDS operations (lgkmcnt) but, unlike __syncthreads(), not for
// outstanding global->LDS loads: callers wait for those explicitly with
// s_waitcnt vmcnt(N) so that later chunks stay in flight across the barrier.
// The wait is the builtin (0xC07F = lgkmcnt(0), other counters unconstrained)
// so that the compiler knows every LDS read before it has completed; the empty
// asm statements keep memory accesses from moving across the barrier.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// LeakyReLU with slope 0.1 as max(v, 0.1 v): the same value as the two-branch
// form for every v (0.1 v <= v exactly when v >= 0), two VALU operations.
__device__ __forceinline__ float leaky(float v) { return fmaxf(v, 0.1f * v); }

// erfc(x) for x >= 0 without branches: the Chebyshev fit of Numerical Recipes
// (Press et al., 2nd ed., sec. 6.2; fractional error below 1.2e-7),
// erfc(x) = t exp(-x^2 + P(t)), t = 1 / (1 + x / 2), P of degree 9.
__device__ __forceinline__ float erfc_pos(float x) {
  const float t = __builtin_amdgcn_rcpf(fmaf(0.5f, x, 1.f));
  float p = 0.17087277f;
  p = fmaf(p, t, -0.82215223f);
  p = fmaf(p, t, 1.48851587f);
  p = fmaf(p, t, -1.13520398f);
  p = fmaf(p, t, 0.27886807f);
  p = fmaf(p, t, -0.18628806f);
  p = fmaf(p, t, 0.09678418f);
  p = fmaf(p, t, 0.37409196f);
  p = fmaf(p, t, 1.00002368f);
  p = fmaf(p, t, -1.26551223f);
  return t * __expf(fmaf(-x, x, p));
}

// Gaussian rate of one symbol, -log2(max(L, 1e-9)),
// L = 1/2 [erfc((|q| - 1/2) / (sigma sqrt2)) - erfc((|q| + 1/2) / (sigma sqrt2))].
// For q = 0, L = 1 - erfc(u) with u = 1 / (2 sigma sqrt2), and the rate is
// -log1p(-erfc(u)) / ln 2, with log1p(v) = log(1 + v) v / ((1 + v) - 1)
// (Goldberg 1991), accurate where L is close to one.  No branches.
__device__ __forceinline__ float symbol_bits(float q, float sigma) {
  const float a = fabsf(q);
  const float inv = 0.70710678118654752f * __builtin_amdgcn_rcpf(sigma);
  const float e1 = erfc_pos(fabsf(a - 0.5f) * inv), e2 = erfc_pos((a + 0.5f) * inv);
  const float L = 0.5f * (e1 - e2);
  const float b1 = -__log2f(fmaxf(L, 1e-9f));
  const float y = 1.f - e2, d = y - 1.f;  // log1p(-e2) = ln(y) (-e2) / d, or -e2 when y rounds to 1
  // (-e2 / d is within an ulp or two of 1: a reciprocal is accurate enough)
  const float l1p = d == 0.f ? -e2 : __logf(y) * (-e2 * __builtin_amdgcn_rcpf(d));
  const float b0 = fminf(-1.44269504088896341f * l1p, 29.8973529f);  // -log2(1e-9)
  return a == 0.f ? b0 : b1;
}

// sigma = max(softplus(s), 0.11).  Where softplus(s) >= 0.11, exp(s) > 0.11,
// so log(1 + exp(s)) loses nothing to the rounding of 1 + exp(s) at fp32.
__device__ __forceinline__ float softplus_sigma(float s) {
  const float sp = s > 20.f ? s : __logf(1.f + __expf(s));
  return fmaxf(sp, 0.11f);
}

// Entropy-coder scales: sigma_j = SMIN (SMAX / SMIN)^(j / (NS - 1)), j < NS.
constexpr int kCoderScales = 64;
constexpr float kCoderSMin = 0.11f;
constexpr float kCoderLogStepInv = 63.0f / 7.7524524f;  // (NS - 1) / ln(SMAX / SMIN), SMAX = 256

// Scale index of sigma: the smallest j with scales[j] >= sigma (NS - 1 if
// none).  The logarithm only seeds the search; the comparisons decide.
__device__ __forceinline__ int coder_scale_index(float sigma, const float* scales) {
  int j = (int)ceilf(__logf(sigma * (1.f / kCoderSMin)) * kCoderLogStepInv);
  j = min(max(j, 0), kCoderScales - 1);
  while (j > 0 && scales[j - 1] >= sigma) --j;
  while (j < kCoderScales - 1 && scales[j] < sigma) ++j;
  return j;
}

// Deterministic (fixed-order) wave reduction of a double.
__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// The frame's rate total, summed by one workgroup of the launch that follows
// the last rate partials on the stream (the launch boundary makes them
// visible): thread t adds elements t, t + blockDim, ... of part[0, n), then
// the waves are added in order, so the sum has a fixed order.  Called
// uniformly by every thread of that workgroup.
__device__ __forceinline__ void block_sum_to(const double* part, int n, double* out) {
  __shared__ double red[16];
  double v = 0.0;
  for (int i = threadIdx.x; i < n; i += blockDim.x) v += part[i];
  v = wave_sum(v);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  if (threadIdx.x == 0) {
    double t = 0.0;
    for (int w = 0; w < (int)(blockDim.x >> 6); ++w) t += red[w];
    *out = t;
  }
  __syncthreads();
}

}  // namespace nc
