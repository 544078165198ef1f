// fp16 DC block (Supp. B.1, LeakyReLU form) for C = 256 with 64 pixels per
// wave: one wave per SIMD, so every weight fragment a wave reads from LDS
// feeds two MFMAs (two 32-pixel halves) instead of one.
//
// A workgroup of 4 waves owns an 8 x 16 pixel tile.  Wave w = (pg, hf):
// pixel group pg = w & 1 holds tile rows 4 pg .. 4 pg + 3 (64 pixels, two
// halves of two rows each); hf = w >> 1 picks the half of the pw2 output
// channels the wave accumulates, and the parity of the hidden chunks it
// produces.  The 2C = 512 hidden channels are 16 chunks of 32; iteration i
// (8 iterations) handles chunks 2i and 2i + 1: each wave runs the pw1 chain of
// chunk 2i + hf for its 64 pixels (bias start, 16 k-steps, two accumulators),
// applies the LeakyReLU, hands the fp16 result to its partner wave (same
// pixels, other hf) through LDS, and projects both chunks onto its 128 output
// channels.  Every SIMD does the same MFMA work in every iteration.
//
// Weights stream from the chunk-major image of the fp16 block (per chunk: 16
// pw1 fragments, one bias fragment, 16 pw2 fragments, 1 KiB each) with direct
// global->LDS loads into two pw1 slots and two pw2 slots (two chunks each), a
// phase ahead of their use.
#include <type_traits>

#include "common.hpp"
#include "internal.hpp"

namespace nc {

namespace dc64 {
constexpr int C = 256;
constexpr int KS = C / 16;          // 16 k-steps of pw1
constexpr int NCH = 2 * C / 32;     // 16 hidden chunks
constexpr int NIT = NCH / 2;        // 8 iterations (two chunks each)
constexpr int FR = KS + 1 + 2 * (C / 32);  // 33 fragments per chunk in the image
constexpr int TH = 8, TW = 16;      // tile rows x columns at 1/8 scale
// LDS map (bytes)
constexpr int OW1 = 0;              // pw1 slots: [slot 2][chunk parity 2][k-step 16] x 1 KiB
constexpr int OW2 = 64 * 1024;      // pw2 slots: [slot 2][chunk parity 2][tile 8][k-step 2] x 1 KiB
constexpr int OHID = 128 * 1024;    // hidden hand-off: [buffer 2][wave 4][half 2][k-step 2] x 1 KiB
constexpr int SMEM = 160 * 1024;
// set-up: wave (pg, hf)'s halo band (rows 4 pg - 1 .. 4 pg + 4 of the tile,
// 18 columns, channels 128 hf .. + 127: 256 bytes per pixel) in region w,
// later its depthwise outputs in MFMA B-fragment order; the biases pass
// through the end of the hand-off area, which the regions leave free
constexpr int OREG = 32 * 1024;
constexpr int BAND_PX = (TH / 2 + 2) * (TW + 2);  // 108
constexpr int REG = BAND_PX * 256;                // 27 KiB
constexpr int BAND_INSTR = REG / 1024;            // 27 direct loads
constexpr int XF = 1024 + 16;                     // exchange fragment stride
constexpr int OBIAS = SMEM - 3 * 1024;            // 2C + C fp32
static_assert(OREG + 4 * REG <= OBIAS && OBIAS >= OHID, "band regions stay below the biases");
static_assert(16 * XF <= REG, "the exchange fits a region");
static_assert(OHID + 32 * 1024 == SMEM && SMEM <= 160 * 1024, "fits the LDS of a CU");
}  // namespace dc64

// A workgroup of 4 waves owns an 8 x 16 pixel tile.  Wave w = (pg, hf):
// pixel group pg = w & 1 holds tile rows 4 pg .. 4 pg + 3 (64 pixels, two
// halves of two rows each); hf = w >> 1 picks the half of the pw2 output
// channels the wave accumulates, and the parity of the hidden chunks it
// produces: the 2C = 512 hidden channels are 16 chunks of 32, and in
// iteration i each wave runs the pw1 chain of chunk 2 i + hf for its 64
// pixels.  The pipeline runs 9 phases separated by one barrier each: phase i
// runs the chains of iteration i interleaved with the projection of iteration
// i - 1 (both chunks 2 i - 2, 2 i - 1 onto the wave's 128 output channels,
// from the LDS copies of its own hidden chunk and its partner's -- same
// pixels, other hf), so the MFMA pipe always has independent work while
// fragment reads are in flight.  Hidden chunks are handed off through two LDS buffers
// (by phase parity); pw1 and pw2 fragments stream through two slots each,
// loaded one phase ahead.
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void k_dcblock64_f16(BlockArgs a) {
  using namespace dc64;
  __shared__ __attribute__((aligned(1024))) char smem[SMEM];
  const int tiles_x = (a.w + TW - 1) / TW;
  const int ntile = tiles_x * ((a.h + TH - 1) / TH);
  const int tile = xcd_tile(blockIdx.x, gridDim.x);
  if (tile >= ntile) return;
  const int ty0 = (tile / tiles_x) * TH, tx0 = (tile % tiles_x) * TW;
  const int lane = threadIdx.x & 63, h = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int pg = wave & 1, hf = wave >> 1;
  const f16* z = (const f16*)a.src;
  const char* wimg = (const char*)a.w1;

  // chunk j's pw1 part (fragments 0 .. 15) or pw2 part (17 .. 32), 4 fragments per wave
  auto issue_part = [&](int j, bool pw2, char* dst) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int f = wave + 4 * i;
      dma16(wimg + ((size_t)j * FR + (pw2 ? KS + 1 : 0) + f) * 1024 + lane * 16, dst + f * 1024);
    }
  };
  // the m-th of this wave's 4 direct loads of chunk j's pw1 or pw2 part
  auto issue_one = [&](int j, bool pw2, char* dst, int m) __attribute__((always_inline)) {
    const int f = wave + 4 * m;
    dma16s(wimg + ((size_t)j * FR + (pw2 ? KS + 1 : 0) + f) * 1024, (uint32_t)lane * 16, dst + f * 1024);
  };
  auto w1slot = [&](int slot, int cp) __attribute__((always_inline)) { return smem + OW1 + (2 * slot + cp) * 16384; };
  auto w2slot = [&](int slot, int cp) __attribute__((always_inline)) { return smem + OW2 + (2 * slot + cp) * 16384; };
  auto hid = [&](int buf, int w_) __attribute__((always_inline)) { return (half8*)(smem + OHID + buf * 16384 + w_ * 4096); };

  // ---- set-up: biases, halo band, chunks 0 and 1 (pw1), depthwise, exchange
  // depthwise role: channels 128 hf + 2 cp, +1 (cp = lane) for the 4 x 16
  // pixels of group pg; the wave's band holds exactly its residual too
  const int cp = lane;
  const int c0 = 128 * hf + 2 * cp;
  half2 wt[9];
  float bias0, bias1;
  {
    const intx4* wsrc = (const intx4*)a.dww + 3 * (c0 / 2);
    intx4 q0 = wsrc[0], q1 = wsrc[1];
    intx3 q2 = *(const intx3*)(wsrc + 2);
    // consumed here, before the direct loads are issued, so that the
    // compiler's wait for them does not also wait for those loads
    asm volatile("" : "+v"(q0), "+v"(q1), "+v"(q2));
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
  char* const own = smem + OREG + wave * REG;
  // biases (2C + C fp32 = 3 KiB), wave 0
  if (wave == 0) {
    dma16((const char*)a.b1 + lane * 16, smem + OBIAS);
    dma16((const char*)a.b1 + 1024 + lane * 16, smem + OBIAS + 1024);
    dma16((const char*)a.b2 + lane * 16, smem + OBIAS + 2048);
  }
  // band: unit S of the region is 16-byte unit S % 16 of halo pixel S / 16
#pragma unroll
  for (int i = 0; i < BAND_INSTR; ++i) {
    const int S = i * 64 + lane;
    const int hp = S >> 4, u = S & 15;
    const int hy = ty0 + 4 * pg - 1 + hp / (TW + 2), hx = tx0 - 1 + hp % (TW + 2);
    const bool in = hy >= 0 && hy < a.h && hx >= 0 && hx < a.w;
    dma16(in ? z + (size_t)(hy * a.w + hx) * C + 128 * hf + 8 * u : (const f16*)a.zpad, own + i * 1024);
  }
  // chunks 0 and 1, pw1 part, into slot 0 (the depthwise does not touch it)
  issue_part(0, false, w1slot(0, 0));
  issue_part(1, false, w1slot(0, 1));
  // The depthwise runs row by row as the band arrives: output row r needs band
  // rows r .. r + 2, and band row y is complete once direct load (18 y + 17) / 4
  // has landed (4 halo pixels per load).  The loads return in order, so
  // "rows up to y in" is "at most 26 - (18 y + 17) / 4 band loads and the 8
  // chunk loads still outstanding" (the biases, issued first, are in too).
  // Band rows as tap pairs of one channel, P0[y][x] = (z[y][x], z[y][x + 1]) of
  // channel c0 and P1 of channel c1 (x = 0 .. 16, one byte permute each), so
  // that every v_dot2_f32_f16 takes two taps of a row: (w0, w1) . (z[k],
  // z[k + 1]) and (0, w2) . (z[k + 1], z[k + 2]), accumulated in fp32.
  half2 P0[TH / 2 + 2][TW + 1], P1[TH / 2 + 2][TW + 1];
  auto load_row = [&](int y) __attribute__((always_inline)) {
    uint32_t vr[TW + 2];
#pragma unroll
    for (int x = 0; x < TW + 2; ++x) vr[x] = *(const uint32_t*)(own + (y * (TW + 2) + x) * 256 + cp * 4);
#pragma unroll
    for (int x = 0; x < TW + 1; ++x) {
      P0[y][x] = __builtin_bit_cast(half2, __builtin_amdgcn_perm(vr[x + 1], vr[x], 0x05040100u));
      P1[y][x] = __builtin_bit_cast(half2, __builtin_amdgcn_perm(vr[x + 1], vr[x], 0x07060302u));
    }
  };
  half2 W0a[3], W0b[3], W1a[3], W1b[3];
#pragma unroll
  for (int ky = 0; ky < 3; ++ky) {
    W0a[ky] = half2{wt[3 * ky][0], wt[3 * ky + 1][0]};
    W0b[ky] = half2{(f16)0.f, wt[3 * ky + 2][0]};
    W1a[ky] = half2{wt[3 * ky][1], wt[3 * ky + 1][1]};
    W1b[ky] = half2{(f16)0.f, wt[3 * ky + 2][1]};
  }
  // The residual of this wave's outputs (the band's interior), kept in
  // registers until the epilogue as the B operand of the identity MFMAs: for
  // output tile t, half hh, step q, lane = (pixel p = 32 hh + lane % 32,
  // channel unit 4 t + 2 q + lane / 32 of the wave's 128 channels).  Half hh
  // lies in band rows 2 hh + 1, 2 hh + 2, read before the depthwise outputs
  // overwrite them.
  half8 res[4][2][2];
  auto load_res = [&](int hh) __attribute__((always_inline)) {
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const int p = 32 * hh + (lane & 31);
        const int hp = ((p >> 4) + 1) * (TW + 2) + (p & 15) + 1;
        res[t][hh][q] = *(const half8*)(own + hp * 256 + (4 * t + 2 * q + h) * 16);
      }
  };
  // output (row r of the group, column x) of channel pair cp goes to the B
  // fragment of half r / 2, k-step 8 hf + cp / 8: fragment index
  // 8 (r / 2) + cp / 8 of this region, lane 16 (r % 2) + x + 32 ((cp / 4) % 2),
  // element 2 (cp % 4).  Rows 0, 1 write bytes [0, 8 XF) of the region (band
  // rows 0, 1, consumed), rows 2, 3 bytes [8 XF, 16 XF) (band rows 1 .. 3,
  // consumed by then).
  const int xhalf = (cp >> 2) & 1;
  auto dw_row = [&](int r) __attribute__((always_inline)) {
#pragma unroll
    for (int k = 0; k < TW; ++k) {
      float a0 = bias0, a1 = bias1;
#pragma unroll
      for (int ky = 0; ky < 3; ++ky) {
        a0 = __builtin_amdgcn_fdot2(W0a[ky], P0[r + ky][k], a0, false);
        a0 = __builtin_amdgcn_fdot2(W0b[ky], P0[r + ky][k + 1], a0, false);
        a1 = __builtin_amdgcn_fdot2(W1a[ky], P1[r + ky][k], a1, false);
        a1 = __builtin_amdgcn_fdot2(W1b[ky], P1[r + ky][k + 1], a1, false);
      }
      half2 o;
      o[0] = (f16)a0;
      o[1] = (f16)a1;
      const int f = 8 * (r >> 1) + (cp >> 3);
      const int px = 16 * (r & 1) + k;
      *(half2*)(own + f * XF + (px + 32 * xhalf) * 16 + (cp & 3) * 4) = o;
    }
  };
  static_assert(BAND_INSTR == 27 && (18 * 5 + 17) / 4 == 26, "band row -> load index");
  asm volatile("s_waitcnt vmcnt(21)" ::: "memory");  // band rows 0 .. 2
  load_row(0);
  load_row(1);
  load_row(2);
  load_res(0);
  dw_row(0);
  asm volatile("s_waitcnt vmcnt(17)" ::: "memory");  // band row 3
  load_row(3);
  dw_row(1);
  asm volatile("s_waitcnt vmcnt(12)" ::: "memory");  // band row 4
  load_row(4);
  load_res(1);
  dw_row(2);
  asm volatile("s_waitcnt vmcnt(8)" ::: "memory");  // band row 5
  load_row(5);
  dw_row(3);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // chunks 0, 1 (pw1) too
  lds_barrier();

  // pw1 operand: all C filtered channels of this wave's 64 pixels
  half8 av[2][KS];
#pragma unroll
  for (int hh = 0; hh < 2; ++hh)
#pragma unroll
    for (int s = 0; s < KS; ++s)
      av[hh][s] = *(const half8*)(smem + OREG + (pg + 2 * (s >> 3)) * REG + (8 * hh + (s & 7)) * XF + lane * 16);
  // pw2 accumulators of this wave's 4 output tiles (channels 128 hf + 32 t ..)
  // for both halves, starting from the bias
  floatx16 out[4][2];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int tt = 4 * hf + t;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const floatx4 bv = *(const floatx4*)(smem + OBIAS + 2048 + (32 * tt + 8 * g + 4 * h) * 4);
#pragma unroll
      for (int e = 0; e < 4; ++e) out[t][0][4 * g + e] = out[t][1][4 * g + e] = bv[e];
    }
  }
  // pw1 biases of the chunks this wave produces, as the A operand of one MFMA
  // against a one-hot B: lane l < 32 holds the bias of row l at k = 0, so the
  // product is the bias broadcast over the 32 pixel columns (exact in fp32)
  f16 b1v[NIT];
#pragma unroll
  for (int i = 0; i < NIT; ++i) b1v[i] = (f16)((const float*)(smem + OBIAS))[32 * (2 * i + hf) + (lane & 31)];
  lds_barrier();  // the regions and the bias copies are dead from here on
  half8 ones = {};
  ones[0] = (f16)(lane < 32 ? 1.f : 0.f);


  auto phase = [&](auto ic) __attribute__((always_inline)) {
    constexpr int i = decltype(ic)::value;
    constexpr bool CHAIN = i < NIT, PROJ = i > 0;
    floatx16 hacc[2];
    // hidden chunks of iteration i - 1, [half][k-step]: this wave's (gx), read
    // at the start, and the partner's (gy), read during the first half
    half8 gx[2][2];
    half8 gy[2][2];
    if constexpr (PROJ) {
#pragma unroll
      for (int hh = 0; hh < 2; ++hh)
#pragma unroll
        for (int u = 0; u < 2; ++u) gx[hh][u] = hid((i - 1) & 1, wave)[(2 * hh + u) * 64 + lane];
    }
    // chain fragment s: pw1 k-step s of chunk 2 i + hf; projection fragment s:
    // s < 8 this wave's chunk, else the partner's, (tile t, k-step u) = s % 8
    const half8* w1 = (const half8*)w1slot(i & 1, hf) + lane;
    const half8* wo = (const half8*)w2slot((i - 1) & 1, hf) + lane + 8 * hf * 64;
    const half8* wp = (const half8*)w2slot((i - 1) & 1, hf ^ 1) + lane + 8 * hf * 64;
    auto w2at = [&](int s) __attribute__((always_inline)) { return (s < 8 ? wo : wp)[(s & 7) * 64]; };
    // rolling window: the reads for step s + PF are issued before the MFMAs of
    // step s, so each read has PF steps of MFMA work to land in (one wave per
    // SIMD hides the LDS latency itself); sched_barrier keeps the order
    constexpr int PF = 3;
    half8 q1[PF], q2[PF];
#pragma unroll
    for (int s = 0; s < PF; ++s) {
      if constexpr (CHAIN) q1[s] = w1[s * 64];
      if constexpr (PROJ) q2[s] = w2at(s);
    }
    if constexpr (CHAIN) {
      half8 ab = {};
      ab[0] = lane < 32 ? b1v[i] : (f16)0.f;
      hacc[0] = mfma_f16(ab, ones, floatx16{});
      hacc[1] = mfma_f16(ab, ones, floatx16{});
    }
    __builtin_amdgcn_sched_barrier(0);
    // The projection runs LAG steps behind the chain, so that the chain's
    // LeakyReLU and hand-off overlap the last projection MFMAs instead of
    // waiting for the pipe to drain.  LAG = 1 measured best (31 shader clocks
    // per MFMA over the loop at 1080p, against 32 for the MFMA itself); with
    // LAG >= 3 the register allocation needs more copies and the loop takes
    // about 40 % longer.
    constexpr int LAG = CHAIN && PROJ ? 1 : 0;
    half8 g[2][2];
    auto leaky_part = [&](int k) __attribute__((always_inline)) {
      // LeakyReLU of the fp16-rounded hidden values, max(h, 0.1 h) in packed
      // fp16, as B fragment (half k >> 1, k-step k & 1) (the pw2 weights are
      // packed in this register order); handed to the partner.  Packed fp16
      // halves the VALU work of the step that cannot overlap the MFMAs (6 %
      // of the loop); the result is within one fp16 unit of rounding
      // max(h, 0.1 h) taken in fp32.  With LAG < 4 the last step does the
      // remaining parts.
      const int hh = k >> 1, u = k & 1;
      half8 hv;
#pragma unroll
      for (int e = 0; e < 8; ++e) hv[e] = (f16)hacc[hh][8 * u + e];
      const half8 sl = hv * (f16)0.1f;
#pragma unroll
      for (int e = 0; e < 8; ++e) g[hh][u][e] = __builtin_fmaxf16(hv[e], sl[e]);
      hid(i & 1, wave)[(2 * hh + u) * 64 + lane] = g[hh][u];
    };
#pragma unroll
    for (int s = 0; s < 16 + LAG; ++s) {
      const int c = s, pj = s - LAG;  // chain step, projection step
      const bool dc = CHAIN && c < 16, dp = PROJ && pj >= 0 && pj < 16;
      half8 a1, a2;
      if (dc) {
        a1 = q1[c % PF];
        if (c + PF < 16) q1[c % PF] = w1[(c + PF) * 64];
      }
      if (dp) {
        a2 = q2[pj % PF];
        if (pj + PF < 16) q2[pj % PF] = w2at(pj + PF);
      }
      if (dc) {
        hacc[0] = mfma_f16(a1, av[0][c], hacc[0]);
        hacc[1] = mfma_f16(a1, av[1][c], hacc[1]);
      }
      if (dp) {
        const int t = (pj & 7) >> 1, u = pj & 1;
        const half8 b0 = pj < 8 ? gx[0][u] : gy[0][u], b1 = pj < 8 ? gx[1][u] : gy[1][u];
        out[t][0] = mfma_f16(a2, b0, out[t][0]);
        out[t][1] = mfma_f16(a2, b1, out[t][1]);
      }
      if (PROJ && pj == 4) {  // the partner's hidden chunk, four steps before its use
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
#pragma unroll
          for (int u = 0; u < 2; ++u) gy[hh][u] = hid((i - 1) & 1, wave ^ 2)[(2 * hh + u) * 64 + lane];
      }
      if (CHAIN && LAG > 0 && c >= 16) {
#pragma unroll
        for (int k = 4 * (c - 16) / LAG; k < 4 * (c - 15) / LAG; ++k) leaky_part(k);
      }
      // the loads into the slots freed by the previous barrier, one per step:
      // pw1 of iteration i + 1 (into the slot of chain i - 1), pw2 of
      // iteration i (into the slot of projection i - 2)
      if (s < 8 && i + 1 < NIT) issue_one(2 * i + 2 + (s >> 2), false, w1slot((i + 1) & 1, s >> 2), s & 3);
      if (s >= 8 && s < 16 && i < NIT) issue_one(2 * i + ((s - 8) >> 2), true, w2slot(i & 1, (s - 8) >> 2), s & 3);
      __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (CHAIN && LAG == 0) {
#pragma unroll
      for (int k = 0; k < 4; ++k) leaky_part(k);
    }
    // this phase's loads have landed (the next phase's fragments), every
    // hand-off is visible, every slot read is done
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    lds_barrier();
  };
  phase(std::integral_constant<int, 0>{});
  phase(std::integral_constant<int, 1>{});
  phase(std::integral_constant<int, 2>{});
  phase(std::integral_constant<int, 3>{});
  phase(std::integral_constant<int, 4>{});
  phase(std::integral_constant<int, 5>{});
  phase(std::integral_constant<int, 6>{});
  phase(std::integral_constant<int, 7>{});
  phase(std::integral_constant<int, 8>{});

  // Epilogue: the residual enters the accumulators through the MFMA (the two
  // 32 x 16 halves of the identity as A, exact in fp32); the
  // sums are rounded once to fp16 and parked (group 0 in pw2 slot 0, group 1
  // in the hand-off area; row = pixel, 8-byte unit u of the row at
  // u ^ (row & 15)), then stored as 16-byte vectors, 8 channels of one pixel
  // per thread.
  auto park = [&](int g) __attribute__((always_inline)) { return smem + (g ? OHID : OW2); };
  {
    const int row = lane & 31;
    half8 e0, e1;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      e0[e] = (f16)(row == 8 * h + e ? 1.f : 0.f);
      e1[e] = (f16)(row == 16 + 8 * h + e ? 1.f : 0.f);
    }
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int hh = 0; hh < 2; ++hh)
#pragma unroll
        for (int q = 0; q < 2; ++q) out[t][hh] = mfma_f16(q ? e1 : e0, res[t][hh][q], out[t][hh]);
    char* ob = park(pg);
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const int p = 32 * hh + row;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int cc = 32 * (4 * hf + t) + 8 * g + 4 * h;
          half4 o;
#pragma unroll
          for (int e = 0; e < 4; ++e) o[e] = (f16)out[t][hh][4 * g + e];
          *(half4*)(ob + p * 512 + (((cc >> 2) ^ (p & 15)) << 3)) = o;
        }
      }
  }
  lds_barrier();
  f16* dst = (f16*)a.dst;
#pragma unroll
  for (int i = 0; i < 128 * 32 / 256; ++i) {
    const int idx = i * 256 + threadIdx.x;
    const int px = idx >> 5, k8 = idx & 31;  // tile pixel, 8-channel unit
    const int g = px >> 6, p = px & 63;
    const int yy = ty0 + (px >> 4), xx = tx0 + (px & 15);
    if (yy < a.h && xx < a.w) {
      const char* ob = park(g) + p * 512;
      // units 2 k8 and 2 k8 + 1 are the aligned pair at 2 k8 ^ (p & 14), swapped when p is odd
      const half8 pv = *(const half8*)(ob + (((2 * k8) ^ (p & 14)) << 3));
      half8 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        o[e] = (p & 1) ? pv[4 + e] : pv[e];
        o[4 + e] = (p & 1) ? pv[e] : pv[4 + e];
      }
      __builtin_nontemporal_store(o, (half8*)(dst + (size_t)(yy * a.w + xx) * C + 8 * k8));
    }
  }
}

hipError_t launch_dcblock64_f16(const BlockArgs& a, hipStream_t st) {
  launch(k_dcblock64_f16, dim3(dc_grid(a.h, a.w)), dim3(256), st, a);
  return hipGetLastError();
}

}  // namespace nc
