// fp16 DC block (Supp. B.1, LeakyReLU and gated forms) for C = 256 with 128 pixels per
// wave: each wave covers the whole 8 x 16 pixel tile of its workgroup, so
// every weight fragment it loads feeds four MFMAs (the tile's four 32-pixel
// groups).  The weight fragments are therefore read straight from global
// memory (L2) into registers as MFMA A operands, never staged through LDS;
// LDS holds only activations: the halo bands, the depthwise result a (the
// pw1 B operand) and the hidden layer (the pw2 B operand).
//
// A workgroup of 4 waves (one per SIMD) owns one tile; 255 tiles at 1080p,
// one per CU.  Wave w owns channel quarter w (64 w .. + 63) of the depthwise
// and of the block's output.
//   1. Depthwise.  Wave w's halo band (10 rows x 18 columns of its 64
//      channels) arrives in LDS by direct global->LDS loads; each output row
//      is filtered as soon as its three band rows are in, accumulated in fp32
//      from the bias with v_dot2_f32_f16 (two taps of a row per instruction),
//      rounded to fp16 once and written as B fragments of a.  The band's
//      interior is the residual of the wave's outputs; it is read into
//      registers before the band's space is reused.
//   2. pw1.  The 2C = 512 hidden channels are 16 chunks of 32; wave w runs
//      the chains of chunks 2 w, 2 w + 1 (round 0) and 8 + 2 w, 9 + 2 w
//      (round 1) over all 128 pixels: 16 k-steps of 8 MFMAs (2 chunks x 4
//      pixel groups) from the bias, LeakyReLU on the fp16-rounded value, the
//      result written as pw2 B fragments (round 0 over the bands, round 1
//      over a once every wave is done with a).
//   3. pw2.  Wave w accumulates output channels 64 w .. + 63 (two 32-row
//      tiles) from the bias plus the residual (added through identity MFMAs,
//      exact products) over all 512 hidden channels (32 k-steps of 8 MFMAs);
//      the sums are rounded to fp16 once, parked in LDS and stored as
//      16-byte vectors.
// The weight fragments of the three loops form one stream of 64 steps (two
// fragments per step), prefetched a fixed number of steps ahead across the
// loop boundaries; the first ones are requested before the halo band.
#include <utility>

#include "common.hpp"
#include "internal.hpp"

namespace nc {

namespace dcw {
constexpr int C = 256;
constexpr int KS = C / 16;                 // 16 k-steps of pw1
constexpr int FR = KS + 1 + 2 * (C / 32);  // 33 fragments per hidden chunk in the weight image
constexpr int TH = 8, TW = 16;             // tile rows x columns at 1/8 scale
constexpr int XF = 1024 + 16;              // LDS stride of one B fragment
// wave w's halo band: rows -1 .. 8, columns -1 .. 16 of the tile, channels
// 64 w .. + 63, 128 bytes per pixel (16-byte unit u of band column x at
// position u ^ bswz(x)); the last direct load runs half past the band
constexpr int BH = TH + 2, BW = TW + 2;            // 10 x 18
constexpr int BROW = BW * 128;                     // bytes per band row
constexpr int BAND_INSTR = (BH * BW * 8 + 63) / 64;  // 23 direct loads of 1 KiB
constexpr int REG = BAND_INSTR * 1024;
constexpr int OA = 4 * REG;                        // a: [group 4][k-step 16] fragments, later the round-1 hidden layer
constexpr int OBIAS = OA + 64 * XF;                // pw1 biases (2C fp32), then pw2 biases (C fp32)
constexpr int SMEM = OBIAS + 3 * C * 4;
static_assert(SMEM <= 160 * 1024, "fits the LDS of a CU");
static_assert(64 * XF <= OA && TH * TW * C * 2 <= OA, "the round-0 hidden layer and the parked output fit over the bands");
// direct load holding the last unit of band row y (loads land in order)
constexpr int band_row_load(int y) { return (8 * (BW * y + BW - 1) + 7) / 64; }
static_assert(band_row_load(BH - 1) == BAND_INSTR - 1, "band geometry");
}  // namespace dcw

// Unit swizzle of band column x: units of neighbouring columns (and of the
// two lane halves' pixels) spread over all LDS banks.
__device__ __forceinline__ constexpr int bswz(int x) { return (x >> 1) & 7; }
// Position of lane slot L (pixel column n = L % 32 = 16 rho + x, k half
// kh = L / 32) inside a 1 KiB B fragment.  Two access patterns must both stay
// free of LDS bank conflicts: the MFMA operand reads and the hidden-layer
// writes (16 bytes per lane, 16 lanes at a time: position mod 16 must be a
// bijection of x for fixed rho, kh), and the depthwise's writes (4 bytes per
// lane; at one output step the lanes write columns x and 15 - x for both k
// halves into 4 consecutive fragments, so those four positions must fall in
// different 4-bank groups mod 16, four apart).  With kk = min(x, 15 - x) and
// side = x > 7: position = 16 (rho + 2 kh) + 4 ((2 (kk / 4) + side + 2 kh) mod 4)
// + kk mod 4.
__device__ __forceinline__ constexpr int bslot(int L) {
  const int rho = (L >> 4) & 1, x = L & 15, kh = L >> 5;
  const int kk = x < 8 ? x : 15 - x, side = x > 7 ? 1 : 0;
  return 16 * (rho + 2 * kh) + 4 * ((2 * (kk >> 2) + side + 2 * kh) & 3) + (kk & 3);
}
// a's fragment (pixel group g, k-step s), later the round-1 hidden fragment
__device__ __forceinline__ constexpr int a_off(int g, int s) { return dcw::OA + (16 * g + s) * dcw::XF; }
// round-0 hidden fragment (g, k), over the bands
__device__ __forceinline__ constexpr int h0_off(int g, int k) { return (16 * g + k) * dcw::XF; }

// f(integral_constant<int, T>) for every T of the sequence, in order
template <typename F, int... T>
__device__ __forceinline__ void unrolled(F& f, std::integer_sequence<int, T...>) {
  (f(std::integral_constant<int, T>{}), ...);
}

// GATED: the gated form (Supp. B.1, WSiLU and Chunk).  Its weight image pairs
// the entries: entry 2 p holds the pw1 fragments of h1 rows 32 p .. +31,
// entry 2 p + 1 those of the matching h2 rows and the pw2 fragments of gated
// channels 32 p .. +31.  Round r's two chains of wave w are then h1 and h2 of
// gated pair 4 r + w, and the hand-off writes g = WSiLU(h1) h2 (32 channels,
// two k-steps) instead of the LeakyReLU of two chunks; pw2 contracts C = 256
// gated channels (16 k-steps) instead of 2C.
//
// CHAIN: blocks 0 .. nb - 1 of a transform in one launch (blk[b] reads
// blk[b - 1].dst).  Each tile keeps its block output in LDS, written straight
// into the next block's band interior, so between blocks only the ring of the
// band (the neighbours' edge pixels) moves through memory: a block other than
// the last stores only the tile's 44 edge pixels, then publishes its progress
// in flags[tile]; the next block waits until every neighbouring tile has
// published that block, then reads its ring (edge stores, ring loads and the
// progress words are device-coherent accesses; the stores' acknowledgements
// are awaited before the word is written).  Every tile of the grid must be
// resident at once (one workgroup per CU; the host checks the occupancy), and
// each wait gives up after a bounded time, recording it in *status.  flags
// hold a running count: every launch adds nb - 1 to each tile's word, so all
// words are equal between launches and a launch reads its base from its own
// tile's word.

// 16-byte device-coherent accesses (the sc1 policy of device-scope atomics:
// past this XCD's L2 to the device's point of coherence), whole 128-byte lines
// per 8 lanes, without a cache-wide fence (a fence would write back or drop
// the whole L2, weights included).  The load's result may only be used after
// wait_coherent() on it.
__device__ __forceinline__ half8 load_coherent16(const f16* p) {
  half8 v;
  asm volatile("global_load_dwordx4 %0, %1, off sc1" : "=v"(v) : "v"(p) : "memory");
  return v;
}
__device__ __forceinline__ void store_coherent16(f16* p, half8 v) {
  asm volatile("global_store_dwordx4 %0, %1, off sc1" ::"v"(p), "v"(v) : "memory");
}

// The 2x2 stride-2 downsample of a tile's block output, parked in LDS (row =
// tile pixel, 8-byte unit u of the row at u ^ (p & 15)): output rows
// 64 w .. + 63 (tiles c = 0, 1) of the tile's 32 latent pixels (4 x 8 at
// 1/16), K = 4C with k = (2 i + j) C + c from pixel (2 Y + i, 2 X + j) (Fig. 4's
// downsampling to 1/16), the k-steps in order from zero, then the fp32 bias
// and one rounding to fp16: the arithmetic of the downsample launch, so the
// result is the same bit for bit.
__device__ __forceinline__ void dc128_down(const char* smem, const DcChainArgs& ca, const BlockArgs& a, int ty0,
                                           int tx0, int wave, int lane) {
  using namespace dcw;
  constexpr int DK = 4 * C / 16;  // 64 k-steps
  const int h = lane >> 5, n = lane & 31, ly = n >> 3, lx = n & 7;
  const half8* wimg = (const half8*)ca.down_w + lane;  // fragment (row tile mt, k-step s) at [(mt DK + s) 64]
  auto afrag = [&](int s, int c) __attribute__((always_inline)) {
    return wimg[((size_t)(2 * wave + c) * DK + s) * 64];
  };
  // B of k-step s: channels 16 (s % 16) + 8 h .. + 7 of tap s / 16 at tile pixel p
  auto bfrag = [&](int s) __attribute__((always_inline)) {
    const int tap = s >> 4;
    const int p = 16 * (2 * ly + (tap >> 1)) + 2 * lx + (tap & 1);
    const int u = 4 * (s & 15) + 2 * h;
    const char* pb = smem + p * 512;
    const half4 lo = *(const half4*)(pb + ((u ^ (p & 15)) << 3));
    const half4 hi = *(const half4*)(pb + (((u + 1) ^ (p & 15)) << 3));
    half8 v;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[e] = lo[e];
      v[4 + e] = hi[e];
    }
    return v;
  };
  constexpr int PD = 8;  // prefetch distance (k-steps) of the weight fragments (registers are free here)
  half8 qa[PD][2];
#pragma unroll
  for (int s = 0; s < PD; ++s)
#pragma unroll
    for (int c = 0; c < 2; ++c) qa[s][c] = afrag(s, c);
  floatx16 acc[2] = {floatx16{}, floatx16{}};
#pragma unroll
  for (int s = 0; s < DK; ++s) {
    const half8 B = bfrag(s);
    half8 A[2];
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      A[c] = qa[s % PD][c];
      if (s + PD < DK) qa[s % PD][c] = afrag(s + PD, c);
    }
#pragma unroll
    for (int c = 0; c < 2; ++c) acc[c] = mfma_f16(A[c], B, acc[c]);
  }
  // latent pixel (Y, X) lies in the image when its top-left child does (the
  // 1/8 sizes are even)
  const int Y = (ty0 >> 1) + ly, X = (tx0 >> 1) + lx;
  if (2 * Y < a.h && 2 * X < a.w) {
    f16* y = (f16*)ca.down_y + (size_t)(Y * (a.w >> 1) + X) * C;
    const float* bias = (const float*)ca.down_b;
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int ch = 64 * wave + 32 * c + 8 * q + 4 * h;
        const floatx4 bv = *(const floatx4*)(bias + ch);
        half4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = (f16)(acc[c][4 * q + e] + bv[e]);
        *(half4*)(y + ch) = o;
      }
  }
}

// One block of a tile (FIRST: its band comes whole from a.src; LAST: its
// output goes whole to a.dst, or with ca->down_w set through the fused
// downsample to ca->down_y; otherwise the chain's ring and edge exchange).
template <bool GATED, bool CHAIN, bool FIRST, bool LAST>
__device__ __forceinline__ void dc128_block(char* smem, const BlockArgs& a, int b, int tile, int tiles_x, int tiles_y,
                                            int wave0, int base, int* flags, int* status,
                                            const DcChainArgs* ca) {
  using namespace dcw;
  constexpr int KH = GATED ? KS / 2 : KS;  // hidden k-steps per round (the pw2 k-steps of a round)
  constexpr int NT = 2 * KS + 2 * KH;      // weight-stream steps: pw1 rounds 0, 1, pw2
  const int tyi = tile / tiles_x, txi = tile - tyi * tiles_x;
  const int ty0 = tyi * TH, tx0 = txi * TW;
  // the wave index, opaque to the compiler: keeps the weight-stream offsets
  // (scalar, one per step) from being hoisted out of the chain's block loop,
  // where they would all stay live at once
  int wave = wave0;
  asm volatile("" : "+s"(wave));
  // the same for the lane index and everything derived from it (the LDS and
  // global offsets of the unrolled loops)
  int lane = threadIdx.x & 63;
  asm volatile("" : "+v"(lane));
  const int h = lane >> 5;
  const int myslot = bslot(lane) * 16;
  constexpr bool first = FIRST, last = LAST;
  const f16* z = (const f16*)a.src;
  const f16* zpad = (const f16*)a.zpad;
  const half8* wimg = (const half8*)a.w1 + lane;  // fragment (chunk j, f) at [(j FR + f) 64]
  // weight-stream step t, fragment c: pw1 round 0 (t < 16: entry 2 w + c,
  // k-step t), round 1 (t < 32: entry 8 + 2 w + c, k-step t - 16), pw2
  // (k = t - 32: output tile 2 w + c, half k % 2 of the entry holding hidden
  // chunk k / 2: entry k / 2, or 2 (k / 2) + 1 in the gated form)
  auto afrag = [&](int t, int c) __attribute__((always_inline)) {
    int f;
    if (t < 2 * KS) {
      f = (8 * (t >> 4) + 2 * wave + c) * FR + (t & 15);
    } else {
      const int k = t - 2 * KS;
      f = (GATED ? 2 * (k >> 1) + 1 : k >> 1) * FR + KS + 1 + 2 * (2 * wave + c) + (k & 1);
    }
    return wimg[(size_t)f * 64];
  };

  // ---- 1. depthwise: wave w = channels 64 w .. + 63; lane = (channel pair
  // cp, half).  Half 0 filters output columns 0 .. 7 (band columns 0 .. 9),
  // half 1 columns 15 .. 8 (band columns 17 .. 8) in mirrored order with
  // mirrored taps: the halves' band reads are an odd number of columns
  // apart, so they fall in different LDS bank halves.
  constexpr int PA = 3, PB = 2;  // prefetch distances (steps) of the A and B windows
  half8 qa[PA][2];
  half8 res[2][4][2];  // residual: (output tile c, group g, half q) B operands
  {
    const int cp = lane & 31, half = lane >> 5;
    const int c0 = 64 * wave + 2 * cp;
    half2 wt[9];
    float bias0, bias1;
    {
      const intx4* wsrc = (const intx4*)a.dww + 3 * (c0 / 2);
      intx4 q0 = wsrc[0], q1 = wsrc[1];
      intx3 q2 = *(const intx3*)(wsrc + 2);
      // consumed here, before the other loads are issued, so that the
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
    // the first weight fragments, the biases (wave 0), then the band
#pragma unroll
    for (int s = 0; s < PA; ++s)
#pragma unroll
      for (int c = 0; c < 2; ++c) qa[s][c] = afrag(s, c);
    if (wave == 0) {
#pragma unroll
      for (int i = 0; i < 2; ++i) dma16((const char*)a.b1 + i * 1024 + lane * 16, smem + OBIAS + i * 1024);
      dma16((const char*)a.b2 + lane * 16, smem + OBIAS + 2048);
    }
    char* const band = smem + wave * REG;
    auto band_load = [&](int i) __attribute__((always_inline)) {
      const int S = i * 64 + lane;  // band unit: pixel S / 8, position S % 8
      const int bp = S >> 3, u = S & 7;
      const int by = bp / BW, bx = bp - by * BW;
      const int hy = ty0 - 1 + by, hx = tx0 - 1 + bx;
      const bool in = bp < BH * BW && hy >= 0 && hy < a.h && hx >= 0 && hx < a.w;
      dma16(in ? z + (size_t)(hy * a.w + hx) * C + 64 * wave + 8 * (u ^ bswz(bx)) : zpad, band + i * 1024);
    };
    // the band's first BAND_FIRST loads now, the rest after the first output row
    constexpr int BAND_FIRST = 14;
    if (first) {
#pragma unroll
      for (int i = 0; i < BAND_FIRST; ++i) band_load(i);
    }
    // the lane's band reads: column col(i) of a row, its channel pair's dword
    int va[TW / 2 + 2];
#pragma unroll
    for (int i = 0; i < TW / 2 + 2; ++i) {
      const int col = half ? TW + 1 - i : i;
      va[i] = col * 128 + (((cp >> 2) ^ bswz(col)) << 4) + (cp & 3) * 4;
    }
    // taps of a row as dot2 pairs (mirrored for half 1): (A0, A1) . (z[k],
    // z[k + 1]) and (0, A2) . (z[k + 1], z[k + 2]) in the lane's column order
    half2 W0a[3], W0b[3], W1a[3], W1b[3];
#pragma unroll
    for (int ky = 0; ky < 3; ++ky) {
      const half2 l = half ? wt[3 * ky + 2] : wt[3 * ky], m = wt[3 * ky + 1], r = half ? wt[3 * ky] : wt[3 * ky + 2];
      W0a[ky] = half2{l[0], m[0]};
      W0b[ky] = half2{(f16)0.f, r[0]};
      W1a[ky] = half2{l[1], m[1]};
      W1b[ky] = half2{(f16)0.f, r[1]};
    }
    // output (row r, step k) of the channel pair: column x = k (half 0) or
    // 15 - k (half 1), a's fragment (group r / 2, k-step 4 w + cp / 8), lane
    // slot 16 (r % 2) + x + 32 ((cp / 4) % 2), elements 2 (cp % 4), + 1
    int wa[2][TW / 2];
#pragma unroll
    for (int rho = 0; rho < 2; ++rho)
#pragma unroll
      for (int k = 0; k < TW / 2; ++k) {
        const int x = half ? TW - 1 - k : k;
        wa[rho][k] = a_off(0, 4 * wave + (cp >> 3)) + bslot(16 * rho + x + 32 * ((cp >> 2) & 1)) * 16 + (cp & 3) * 4;
      }
    // band rows as tap pairs of one channel: P0[y][i] = (z[y][i], z[y][i + 1])
    // of channel c0, P1 of c0 + 1, in the lane's column order
    half2 P0[BH][TW / 2 + 1], P1[BH][TW / 2 + 1];
    auto load_row = [&](int y) __attribute__((always_inline)) {
      uint32_t vr[TW / 2 + 2];
#pragma unroll
      for (int i = 0; i < TW / 2 + 2; ++i) vr[i] = *(const uint32_t*)(band + y * BROW + va[i]);
#pragma unroll
      for (int i = 0; i < TW / 2 + 1; ++i) {
        P0[y][i] = __builtin_bit_cast(half2, __builtin_amdgcn_perm(vr[i + 1], vr[i], 0x05040100u));
        P1[y][i] = __builtin_bit_cast(half2, __builtin_amdgcn_perm(vr[i + 1], vr[i], 0x07060302u));
      }
    };
    // one output (row r, step k) of the channel pair, written into a
    auto dw_out = [&](int r, int k) __attribute__((always_inline)) {
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
      *(half2*)(smem + wa[r & 1][k] + 16 * (r >> 1) * XF) = o;
    };
    auto dw_row = [&](int r) __attribute__((always_inline)) {
#pragma unroll
      for (int k = 0; k < TW / 2; ++k) dw_out(r, k);
    };
    if constexpr (first) {
      // output row r needs band rows .. r + 2: wait until at most
      // (issued - 1 - band_row_load(r + 2)) band loads are outstanding
#define DW_WAIT(r, issued) asm volatile("s_waitcnt vmcnt(%0)" ::"n"((issued) - 1 - band_row_load((r) + 2)) : "memory")
      static_assert(BAND_FIRST > band_row_load(2), "the first output row's band rows are requested first");
      DW_WAIT(0, BAND_FIRST);
      load_row(0);
      load_row(1);
      load_row(2);
      dw_row(0);
#pragma unroll
      for (int i = BAND_FIRST; i < BAND_INSTR; ++i) band_load(i);
      DW_WAIT(1, BAND_INSTR);
      load_row(3);
      dw_row(1);
      DW_WAIT(2, BAND_INSTR);
      load_row(4);
      dw_row(2);
      DW_WAIT(3, BAND_INSTR);
      load_row(5);
      dw_row(3);
      DW_WAIT(4, BAND_INSTR);
      load_row(6);
      dw_row(4);
      DW_WAIT(5, BAND_INSTR);
      load_row(7);
      dw_row(5);
      DW_WAIT(6, BAND_INSTR);
      load_row(8);
      dw_row(6);
      DW_WAIT(7, BAND_INSTR);
      load_row(9);
      dw_row(7);
#undef DW_WAIT
      // the residual of the wave's outputs is its band's interior: (c, g, q),
      // lane = pixel 32 g + lane % 32 of the tile (band row 1 + 2 g + n / 16,
      // column 1 + n % 16), unit 4 c + 2 q + lane / 32
      {
        const int n = lane & 31, x = 1 + (n & 15);
        const char* rb = band + (1 + (n >> 4)) * BROW + x * 128;
        const int f = bswz(x) ^ h;
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
          for (int g = 0; g < 4; ++g)
#pragma unroll
            for (int q = 0; q < 2; ++q) res[c][g][q] = *(const half8*)(rb + 2 * g * BROW + ((f ^ (4 * c + 2 * q)) << 4));
      }
    } else {
      // pass 1, before this block's ring is known: the outputs that read only
      // the interior (rows 1 .. 6, steps 1 .. 7 of each half row: band
      // columns 1 .. 16), and the residual
      auto load_inner = [&](int y) __attribute__((always_inline)) {
        uint32_t vr[TW / 2 + 2];
#pragma unroll
        for (int i = 1; i < TW / 2 + 2; ++i) vr[i] = *(const uint32_t*)(band + y * BROW + va[i]);
#pragma unroll
        for (int i = 1; i < TW / 2 + 1; ++i) {
          P0[y][i] = __builtin_bit_cast(half2, __builtin_amdgcn_perm(vr[i + 1], vr[i], 0x05040100u));
          P1[y][i] = __builtin_bit_cast(half2, __builtin_amdgcn_perm(vr[i + 1], vr[i], 0x07060302u));
        }
      };
      load_inner(1);
      load_inner(2);
#pragma unroll
      for (int r = 1; r <= TH - 2; ++r) {
        load_inner(r + 2);
#pragma unroll
        for (int k = 1; k < TW / 2; ++k) dw_out(r, k);
      }
      // the residual of the wave's outputs is its band's interior: (c, g, q),
      // lane = pixel 32 g + lane % 32 of the tile (band row 1 + 2 g + n / 16,
      // column 1 + n % 16), unit 4 c + 2 q + lane / 32
      {
        const int n = lane & 31, x = 1 + (n & 15);
        const char* rb = band + (1 + (n >> 4)) * BROW + x * 128;
        const int f = bswz(x) ^ h;
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
          for (int g = 0; g < 4; ++g)
#pragma unroll
            for (int q = 0; q < 2; ++q) res[c][g][q] = *(const half8*)(rb + 2 * g * BROW + ((f ^ (4 * c + 2 * q)) << 4));
      }
      // the ring, once every neighbouring tile has published block b - 1 (its
      // edge pixels are in a.src): one lane of wave 0 per neighbour polls its
      // word
      if (wave == 0 && lane < 9 && lane != 4) {
        const int ny = tyi + lane / 3 - 1, nx = txi + lane % 3 - 1;
        if (ny >= 0 && ny < tiles_y && nx >= 0 && nx < tiles_x) {
          const int* f = flags + ny * tiles_x + nx;
          for (int spin = 0; __hip_atomic_load(f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < base + b; ++spin) {
            if (spin > (1 << 16)) {  // about 0.1 s (a poll is a memory round trip): give up, record it
              __hip_atomic_store(status, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
              break;
            }
            __builtin_amdgcn_s_sleep(1);
          }
        }
      }
      lds_barrier();
      // the ring (52 pixels: rows -1 and 8, columns -1 and 16 of rows 0 .. 7)
      // through registers; the interior is this tile's previous output
      constexpr int RING = 2 * BW + 2 * TH;
      half8 rv[(RING * 8 + 63) / 64];
      int ro[(RING * 8 + 63) / 64];
#pragma unroll
      for (int i = 0; i < (RING * 8 + 63) / 64; ++i) {
        const int S = i * 64 + lane, r = S >> 3, u = S & 7;
        const int by = r < BW ? 0 : r < 2 * BW ? BH - 1 : 1 + (r - 2 * BW) % TH;
        const int bx = r < BW ? r : r < 2 * BW ? r - BW : (r < 2 * BW + TH ? 0 : BW - 1);
        const int hy = ty0 - 1 + by, hx = tx0 - 1 + bx;
        const bool in = S < RING * 8 && hy >= 0 && hy < a.h && hx >= 0 && hx < a.w;
        // device-coherent loads (they bypass this XCD's L2, which may hold
        // an older copy of the line): the neighbours wrote these pixels in
        // this launch
        rv[i] = load_coherent16(in ? z + (size_t)(hy * a.w + hx) * C + 64 * wave + 8 * u : zpad);
        ro[i] = S < RING * 8 ? by * BROW + bx * 128 + ((u ^ bswz(bx)) << 4) : -1;
      }
      // the loads are opaque to the compiler: wait for them with the values
      // as operands, so nothing reads them earlier
      static_assert((RING * 8 + 63) / 64 == 7, "seven ring loads per lane");
      asm volatile("s_waitcnt vmcnt(0)"
                   : "+v"(rv[0]), "+v"(rv[1]), "+v"(rv[2]), "+v"(rv[3]), "+v"(rv[4]), "+v"(rv[5]), "+v"(rv[6])
                   :
                   : "memory");
#pragma unroll
      for (int i = 0; i < (RING * 8 + 63) / 64; ++i)
        if (ro[i] >= 0) *(half8*)(band + ro[i]) = rv[i];
      // pass 2: the outputs that read the ring, in the same order of taps
      load_row(0);
      load_row(1);
      load_row(2);
      dw_row(0);
#pragma unroll
      for (int r = 1; r <= TH - 2; ++r) {
        load_row(r + 2);
        dw_out(r, 0);
      }
      load_row(TH + 1);
      dw_row(TH - 1);
    }
  }
  // the bias loads of wave 0 (the band waits above cover them on a first block)
  if (!first) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  lds_barrier();  // a complete; every wave holds its residual, the bands are free

  // ---- 2, 3. pw1 (steps 0 .. 31) and pw2 (steps 32 .. 63)
  floatx16 acc[2][4];  // pw1: chunk c, group g; pw2: output tile c, group g
  // accumulators from the biases in LDS: row0[c] = the first row of chain or
  // tile c (pw1: 0 .. 2C - 1, pw2: 2C ..)
  auto init_acc = [&](int row00, int row01) __attribute__((always_inline)) {
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const float* b = (const float*)(smem + OBIAS) + (c ? row01 : row00) + 4 * h;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const floatx4 bv4 = *(const floatx4*)(b + 8 * q);
#pragma unroll
        for (int g = 0; g < 4; ++g)
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[c][g][4 * q + e] = bv4[e];
      }
    }
  };
  // LeakyReLU of the fp16-rounded hidden values, max(h, 0.1 h) in packed
  // fp16, written as pw2 B fragments: chunk c, half u of the round's chunk
  // pair go to k-step 4 w + 2 c + u of the round (the pw2 weights are packed
  // in this register order); off(g, k) places fragment (g, k)
  auto leaky_write = [&](auto off) __attribute__((always_inline)) {
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int g = 0; g < 4; ++g)
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          half8 hv, gv;
#pragma unroll
          for (int e = 0; e < 8; ++e) hv[e] = (f16)acc[c][g][8 * u + e];
          const half8 sl = hv * (f16)0.1f;
#pragma unroll
          for (int e = 0; e < 8; ++e) gv[e] = __builtin_fmaxf16(hv[e], sl[e]);
          *(half8*)(smem + off(g, 4 * wave + 2 * c + u) + myslot) = gv;
        }
  };
  // Gated hand-off: WSiLU(h1) = h1 sigmoid(4 h1) rounded to fp16, then
  // g = WSiLU(h1) h2 rounded to fp16 (h1, h2: the fp32 chains), as pw2 B
  // fragments: half u of the pair goes to k-step 2 w + u of the round
  auto gate_write = [&](auto off) __attribute__((always_inline)) {
#pragma unroll
    for (int g = 0; g < 4; ++g)
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        half8 gv;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float h1 = acc[0][g][8 * u + e];
          const f16 ws = (f16)(h1 / (1.f + __expf(-4.f * h1)));
          gv[e] = (f16)((float)ws * acc[1][g][8 * u + e]);
        }
        *(half8*)(smem + off(g, 2 * wave + u) + myslot) = gv;
      }
  };
  auto handoff = [&](auto off) __attribute__((always_inline)) {
    if constexpr (GATED) gate_write(off);
    else leaky_write(off);
  };
  // pw1 chains of round r: the rows of entries 8 r + 2 w + c
  auto chain_row = [&](int r, int c) __attribute__((always_inline)) {
    return GATED ? c * C + 32 * (4 * r + wave) : 32 * (8 * r + 2 * wave + c);
  };
  // B fragment of step t, group g: a (pw1, k-step t % 16), then the hidden
  // layer (pw2, k-step t - 32: round 0 below 16, round 1 above)
  auto bfrag = [&](int t, int g) __attribute__((always_inline)) {
    int off;
    if (t < 2 * KS) {
      off = a_off(g, t & 15);
    } else {
      const int k = t - 2 * KS;
      off = k < KH ? h0_off(g, k) : a_off(g, k - KH);
    }
    return *(const half8*)(smem + off + myslot);
  };
  init_acc(chain_row(0, 0), chain_row(0, 1));
  half8 qb[PB][4];
#pragma unroll
  for (int s = 0; s < PB; ++s)
#pragma unroll
    for (int g = 0; g < 4; ++g) qb[s][g] = bfrag(s, g);
  __builtin_amdgcn_sched_barrier(0);
  // one step of the weight stream; t is a compile-time constant
  auto step = [&](auto tc) __attribute__((always_inline)) {
    constexpr int t = decltype(tc)::value;
    if constexpr (t == KS) {
      // round 0 done: its hidden fragments over the bands (no reader before
      // the hand-off barrier), then round 1 from its bias
      handoff(h0_off);
      init_acc(chain_row(1, 0), chain_row(1, 1));
    }
    if constexpr (t == 2 * KS) {
      // round 1 done: once every wave is past its last read of a (the MFMAs
      // read their operands at issue), its hidden fragments replace a; the
      // pw2 accumulators start from the bias
      lds_barrier();
      handoff(a_off);
      init_acc(2 * C + 64 * wave, 2 * C + 64 * wave + 32);
      // the residual enters first, through the identity (the two 32 x 16
      // halves as A, exact products); the sums are rounded to fp16 once
      {
        const int row = lane & 31;
        half8 e0, e1;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          e0[e] = (f16)(row == 8 * h + e ? 1.f : 0.f);
          e1[e] = (f16)(row == 16 + 8 * h + e ? 1.f : 0.f);
        }
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
          for (int g = 0; g < 4; ++g)
#pragma unroll
            for (int q = 0; q < 2; ++q) acc[c][g] = mfma_f16(q ? e1 : e0, res[c][g][q], acc[c][g]);
      }
      lds_barrier();
#pragma unroll
      for (int s = 0; s < PB; ++s)
#pragma unroll
        for (int g = 0; g < 4; ++g) qb[s][g] = bfrag(t + s, g);
    }
    half8 A[2], B[4];
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      A[c] = qa[t % PA][c];
      if (t + PA < NT) qa[t % PA][c] = afrag(t + PA, c);
    }
    // the B window restarts after the round-1 hand-off (step 32)
    const bool bnext = t + PB < NT && (t >= 2 * KS || t + PB < 2 * KS);
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      B[g] = qb[t % PB][g];
      if (bnext) qb[t % PB][g] = bfrag(t + PB, g);
    }
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int g = 0; g < 4; ++g) acc[c][g] = mfma_f16(A[c], B[g], acc[c][g]);
    __builtin_amdgcn_sched_barrier(0);
  };
  unrolled(step, std::make_integer_sequence<int, NT>{});

  lds_barrier();  // every wave is done reading the hidden layer
  if (last) {
    // ---- epilogue: one rounding to fp16, parked in LDS from offset 0 (row =
    // tile pixel, 8-byte unit u of the row at u ^ (row & 15)), stored as
    // 16-byte vectors
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int p = 32 * g + (lane & 31);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int cc = 64 * wave + 32 * c + 8 * q + 4 * h;
          half4 o;
#pragma unroll
          for (int e = 0; e < 4; ++e) o[e] = (f16)acc[c][g][4 * q + e];
          *(half4*)(smem + p * 512 + (((cc >> 2) ^ (p & 15)) << 3)) = o;
        }
      }
    lds_barrier();
    if constexpr (CHAIN) {
      if (ca->down_w) {
        dc128_down(smem, *ca, a, ty0, tx0, wave, lane);
        return;
      }
    }
    f16* dst = (f16*)a.dst;
#pragma unroll
    for (int i = 0; i < TH * TW * 32 / 256; ++i) {
      const int idx = i * 256 + threadIdx.x;
      const int px = idx >> 5, k8 = idx & 31;  // tile pixel, 8-channel unit
      const int yy = ty0 + (px >> 4), xx = tx0 + (px & 15);
      if (yy < a.h && xx < a.w) {
        const char* ob = smem + px * 512;
        // units 2 k8 and 2 k8 + 1 are the aligned pair at 2 k8 ^ (px & 14), swapped when px is odd
        const half8 pv = *(const half8*)(ob + (((2 * k8) ^ (px & 14)) << 3));
        half8 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          o[e] = (px & 1) ? pv[4 + e] : pv[e];
          o[4 + e] = (px & 1) ? pv[e] : pv[4 + e];
        }
        __builtin_nontemporal_store(o, (half8*)(dst + (size_t)(yy * a.w + xx) * C + 8 * k8));
      }
    }
  } else {
    // ---- a block of a chain: the output (one rounding to fp16; zero outside
    // the image, the next depthwise's padding) goes into the interior of the
    // wave's own band: pixel (1 + y, 1 + x), 16-byte unit u = 4 c + q, half h
    char* const band = smem + wave * REG;
    // a tile that lies wholly inside the image needs no zeroing (uniform)
    const bool full = ty0 + TH <= a.h && tx0 + TW <= a.w;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int p = 32 * g + (lane & 31), py = p >> 4, px = p & 15;
      char* const pb = band + (1 + py) * BROW + (1 + px) * 128 + 8 * h;
      const int sw = bswz(1 + px);
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          half4 o;
#pragma unroll
          for (int e = 0; e < 4; ++e) o[e] = (f16)acc[c][g][4 * q + e];
          *(half4*)(pb + (((4 * c + q) ^ sw) << 4)) = o;
        }
      if (!full && !(ty0 + py < a.h && tx0 + px < a.w)) {
#pragma unroll
        for (int u = 0; u < 8; ++u) *(half4*)(pb + ((u ^ sw) << 4)) = half4{};
      }
    }
    // the tile's 44 edge pixels (rows 0 and 7, columns 0 and 15), the wave's
    // 64 channels, from the band to memory for the neighbours' rings
    f16* dst = (f16*)a.dst;
    constexpr int EDGE = 2 * TW + 2 * (TH - 2);
#pragma unroll
    for (int i = 0; i < (EDGE * 8 + 63) / 64; ++i) {
      const int S = i * 64 + lane, e = S >> 3, u = S & 7;
      // edge e: row 0 (e < 16), row 7 (e < 32), column 0 of rows 1 .. 6
      // (e < 38), column 15 of rows 1 .. 6
      const int e6 = e - 2 * TW, side = e6 >= TH - 2 ? 1 : 0;
      const int py = e < TW ? 0 : e < 2 * TW ? TH - 1 : 1 + e6 - side * (TH - 2);
      const int px = e < TW ? e : e < 2 * TW ? e - TW : side * (TW - 1);
      const int yy = ty0 + py, xx = tx0 + px;
      if (S < EDGE * 8 && yy < a.h && xx < a.w) {
        const half8 v = *(const half8*)(band + (1 + py) * BROW + (1 + px) * 128 + ((u ^ bswz(1 + px)) << 4));
        store_coherent16(dst + (size_t)(yy * a.w + xx) * C + 64 * wave + 8 * u, v);
      }
    }
    // publish: every wave's edge stores are complete at the device's point of
    // coherence (their acknowledgements counted down) before the tile's word
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    lds_barrier();
    if (threadIdx.x == 0) __hip_atomic_store(flags + tile, base + b + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

template <bool GATED, bool CHAIN>
__device__ __forceinline__ void dc128_body(const BlockArgs* blk, int nb, int* flags, int* status,
                                           const DcChainArgs* ca) {
  using namespace dcw;
  __shared__ __attribute__((aligned(1024))) char smem[SMEM];
  const int tiles_x = (blk[0].w + TW - 1) / TW, tiles_y = (blk[0].h + TH - 1) / TH;
  const int tile = xcd_tile(blockIdx.x, gridDim.x);
  if (tile >= tiles_x * tiles_y) return;
  const int wave0 = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if constexpr (!CHAIN) {
    dc128_block<GATED, false, true, true>(smem, blk[0], 0, tile, tiles_x, tiles_y, wave0, 0, nullptr, nullptr, nullptr);
  } else {
    // nb >= 2: the first block, the middle ones, the last
    const int base = __builtin_amdgcn_readfirstlane(__hip_atomic_load(flags + tile, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
    dc128_block<GATED, true, true, false>(smem, blk[0], 0, tile, tiles_x, tiles_y, wave0, base, flags, status, ca);
    for (int b = 1; b < nb - 1; ++b)
      dc128_block<GATED, true, false, false>(smem, blk[b], b, tile, tiles_x, tiles_y, wave0, base, flags, status, ca);
    dc128_block<GATED, true, false, true>(smem, blk[nb - 1], nb - 1, tile, tiles_x, tiles_y, wave0, base, flags, status,
                                          ca);
  }
}

template <bool GATED>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void k_dcblock128_f16(BlockArgs a) {
  dc128_body<GATED, false>(&a, 1, nullptr, nullptr, nullptr);
}

template <bool GATED>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void k_dcchain128_f16(DcChainArgs ca) {
  dc128_body<GATED, true>(ca.blk, ca.nb, ca.flags, ca.status, &ca);
}

hipError_t launch_dcblock128_f16(bool gated, const BlockArgs& a, hipStream_t st) {
  if (gated) launch(k_dcblock128_f16<true>, dim3(dc_grid(a.h, a.w)), dim3(256), st, a);
  else launch(k_dcblock128_f16<false>, dim3(dc_grid(a.h, a.w)), dim3(256), st, a);
  return hipGetLastError();
}

hipError_t launch_dcchain128_f16(bool gated, const DcChainArgs& ca, hipStream_t st) {
  if (ca.nb < 2 || ca.nb > kMaxChain) return hipErrorInvalidValue;
  const dim3 grid(dc_grid(ca.blk[0].h, ca.blk[0].w));
  if (gated) launch(k_dcchain128_f16<true>, grid, dim3(256), st, ca);
  else launch(k_dcchain128_f16<false>, grid, dim3(256), st, ca);
  return hipGetLastError();
}

// Workgroups of the chain kernel that fit the device at once (one per CU
// with its 160 KiB of LDS); the chain needs every tile resident.
int dcchain128_resident(bool gated) {
  int dev = 0, per_cu = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  const hipError_t e = gated ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_dcchain128_f16<true>, 256, 0)
                             : hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_dcchain128_f16<false>, 256, 0);
  return e == hipSuccess ? per_cu * cus : 0;
}

}  // namespace nc
