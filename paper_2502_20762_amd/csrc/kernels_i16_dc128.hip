// Integer DC block (Supp. B.1, LeakyReLU form; Sec. 4.5 and Supp. B.4, Alg. 1)
// for C = 256 with 128 pixels per wave, on the layout of the fp16 block of the
// same width: a workgroup of 4 waves (one per SIMD) owns an 8 x 16 pixel
// tile, every wave covers the whole tile, so each weight fragment it loads
// feeds four MFMAs (the tile's four 32-pixel groups) and is read straight
// from global memory (L2) into registers as the MFMA A operand; LDS holds
// only activations (halo bands, the depthwise result a, the hidden layer).
//
// Every int16 x int16 contraction is exact on the int8 MFMA with the digit
// split of the integer pointwise kernels (x = 256 xh + xl' + 128,
// w = 256 wh + wl, the 128 sum w term and 512 b pre-added per row as the
// correction).  The three digit sums share one wrapping int32 accumulator,
// taken in Horner order over the whole contraction, in four passes of the
// same shape (two fragments of A, four of B, eight MFMAs per step):
//   acc = sum wh xh;  acc <<= 8;  acc += sum wh xl' + sum wl xh;
//   acc = (acc << 8) + corr;  acc += sum wl xl'
// which is 65536 hh + 256 (hl + lh) + ll + corr modulo 2^32: the exact sum
// whenever that fits int32, as the pointwise kernels' combination.
//   1. Depthwise: wave w = channels 64 w .. + 63 over the whole tile, lane =
//      (channel pair, half row); exact int32 sums with v_dot2_i32_i16 (two
//      taps of a row per instruction) from the bias 512 b, rescaled to int16
//      (clip(RHE(s / 8192))), split into int8 digits and written as the pw1
//      B fragments (the two lanes of a channel quad pair up through DPP: one
//      writes the quad's high digits, the other its low digits).
//   2. pw1: hidden chunks of 32 rows; wave w runs chunks 2 w, 2 w + 1
//      (round 0) and 8 + 2 w, 9 + 2 w (round 1) over all 128 pixels, then
//      rescales, applies the integer LeakyReLU and writes the digits as pw2 B
//      fragments in accumulator-register order (the weight image's pw2
//      contraction index follows that order).
//   3. pw2: wave w accumulates output channels 64 w .. + 63 over the 512
//      hidden channels; the sums are rescaled, the residual is added with
//      saturation, and the result stored.
// The weight image is the integer block's chunk-major one: per hidden chunk
// j, 8 pw1 hi-digit fragments, 8 lo-digit ones, then 8 pw2 hi and 8 lo
// fragments (one per 32-row output tile), 1 KiB each.  Chains of blocks in
// one launch work as in the fp16 block: each tile keeps its output in LDS and
// exchanges only its edge pixels through memory.
#include <utility>

#include "common.hpp"
#include "internal.hpp"

namespace nc {

namespace dciw {
constexpr int C = 256;
constexpr int KSI = C / 32;           // 8 k-steps of 32 channels (pw1)
constexpr int MT = C / 32;            // 8 output tiles of 32 rows (pw2)
constexpr int FR = 2 * KSI + 2 * MT;  // 32 fragments per hidden chunk in the weight image
constexpr int TH = 8, TW = 16;
constexpr int XF = 1024 + 16;  // LDS stride of one B fragment
constexpr int BH = TH + 2, BW = TW + 2;
constexpr int BROW = BW * 128;
constexpr int BAND_INSTR = (BH * BW * 8 + 63) / 64;  // 23 direct loads of 1 KiB
constexpr int REG = BAND_INSTR * 1024;
// a: [group 4][k-step 8][digit 2] fragments, later the round-1 hidden layer
// ([group 4][chunk 8][digit 2]); the round-0 hidden layer lies over the bands
constexpr int OA = 4 * REG;
constexpr int OCORR = OA + 64 * XF;  // pw1 corrections (2C int32), then the pw2 ones (C int32)
constexpr int SMEM = OCORR + 3 * C * 4;
constexpr int NT = 128;  // weight-stream steps: pw1 rounds 0, 1 (4 passes of 8), pw2 (4 passes of 16)
static_assert(SMEM <= 160 * 1024, "fits the LDS of a CU");
static_assert(64 * XF <= OA && TH * TW * C * 2 <= OA, "the round-0 hidden layer and the parked output fit over the bands");
constexpr int band_row_load(int y) { return (8 * (BW * y + BW - 1) + 7) / 64; }
static_assert(band_row_load(BH - 1) == BAND_INSTR - 1, "band geometry");
}  // namespace dciw

namespace {

// Unit swizzle of band column x and the lane-slot permutation of a 1 KiB B
// fragment (lane slot L: pixel column n = L % 32 = 16 rho + x, k half
// kh = L / 32), as in the fp16 block, and free of LDS bank conflicts for the
// same reasons: the hidden-layer writes and the MFMA operand reads are 16
// bytes per lane, and at one depthwise output step the lanes write columns x
// and 15 - x, both k halves, into four consecutive fragments (two k-steps x
// two digits) whose positions fall in different 4-bank groups.
__device__ __forceinline__ constexpr int bswz(int x) { return (x >> 1) & 7; }
__device__ __forceinline__ constexpr int bslot(int L) {
  const int rho = (L >> 4) & 1, x = L & 15, kh = L >> 5;
  const int kk = x < 8 ? x : 15 - x, side = x > 7 ? 1 : 0;
  return 16 * (rho + 2 * kh) + 4 * ((2 * (kk >> 2) + side + 2 * kh) & 3) + (kk & 3);
}
__device__ __forceinline__ constexpr int a_off(int g, int f) { return dciw::OA + (16 * g + f) * dciw::XF; }
__device__ __forceinline__ constexpr int h0_off(int g, int f) { return (16 * g + f) * dciw::XF; }

template <typename F, int... T>
__device__ __forceinline__ void unrolled(F& f, std::integer_sequence<int, T...>) {
  (f(std::integral_constant<int, T>{}), ...);
}

// RHE(a / 8192) for any int32 a, before the saturation to int16 (|a| >= 2^28
// saturates either way, so a is clamped first; then the round-half-even bias
// add stays in range).
__device__ __forceinline__ int rhe13(int a) {
  const int ac = min(max(a, -(1 << 28)), 1 << 28);
  return (ac + 4095 + ((ac >> 13) & 1)) >> 13;
}
// clip(RHE(a / 8192)) to int16 for any int32 a: clamping a to
// [-2^28, 2^28 - 4097] first gives the saturated value directly (every a above
// 2^28 - 4097 rounds to at least 32768, every a below -2^28 to at most -32768,
// and the bounds themselves round to 32767 and -32768).
__device__ __forceinline__ int rescale13c(int a) {
  const int ac = min(max(a, -(1 << 28)), (1 << 28) - 4097);
  return (ac + 4095 + ((ac >> 13) & 1)) >> 13;
}
typedef short short2v __attribute__((ext_vector_type(2)));
// Two int32 values saturated to int16 and packed (first in the low half).
__device__ __forceinline__ uint32_t pack_sat(int lo, int hi) {
  return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pk_i16(lo, hi));
}
// High digits (signed) and low digits offset by -128 of the four int16 values
// of dwords d0 (first two) and d1 (last two).
__device__ __forceinline__ uint32_t digits_hi(uint32_t d0, uint32_t d1) {
  return __builtin_amdgcn_perm(d1, d0, 0x07050301u);
}
__device__ __forceinline__ uint32_t digits_lo(uint32_t d0, uint32_t d1) {
  return __builtin_amdgcn_perm(d1, d0, 0x06040200u) ^ 0x80808080u;
}

__device__ __forceinline__ intx4 load_coherent16i(const int16_t* p) {
  intx4 v;
  asm volatile("global_load_dwordx4 %0, %1, off sc1" : "=v"(v) : "v"(p) : "memory");
  return v;
}
__device__ __forceinline__ void store_coherent16i(int16_t* p, intx4 v) {
  asm volatile("global_store_dwordx4 %0, %1, off sc1" ::"v"(p), "v"(v) : "memory");
}

}  // namespace

// One block of a tile (FIRST: its band comes whole from a.src; LAST: its
// output goes whole to a.dst; otherwise the chain's ring and edge exchange,
// with the progress words and bounded waits of the fp16 chain kernel).
template <bool CHAIN, bool FIRST, bool LAST>
__device__ __forceinline__ void dci128_block(char* smem, const BlockArgs& a, int b, int tile, int tiles_x, int tiles_y,
                                             int wave0, int base, int* flags, int* status) {
  using namespace dciw;
  const int tyi = tile / tiles_x, txi = tile - tyi * tiles_x;
  const int ty0 = tyi * TH, tx0 = txi * TW;
  // wave and lane opaque to the compiler: keeps the per-step offsets from
  // being hoisted out of a chain's block loop
  int wave = wave0;
  asm volatile("" : "+s"(wave));
  int lane = threadIdx.x & 63;
  asm volatile("" : "+v"(lane));
  const int h = lane >> 5;
  const int myslot = bslot(lane) * 16;
  constexpr bool first = FIRST, last = LAST;
  const int16_t* z = (const int16_t*)a.src;
  const int16_t* zpad = (const int16_t*)a.zpad;
  const intx4* wimg = (const intx4*)a.w1 + lane;  // fragment f at [f 64]
  // step t, fragment c: pw1 (t < 64: round r = t / 32, pass p = (t / 8) % 4,
  // k-step t % 8 of chunk 8 r + 2 w + c) or pw2 (pass p = (t - 64) / 16,
  // hidden chunk (t - 64) % 16, output tile 2 w + c); passes take the A digit
  // p / 2 (hi, hi, lo, lo) and the B digit p % 2 (hi, lo, hi, lo)
  auto afrag = [&](int t, int c) __attribute__((always_inline)) {
    int f;
    if (t < 64) {
      const int p = (t >> 3) & 3, j = 8 * (t >> 5) + 2 * wave + c;
      f = j * FR + (p >> 1) * KSI + (t & 7);
    } else {
      const int u = t - 64, p = u >> 4, j = u & 15;
      f = j * FR + 2 * KSI + (p >> 1) * MT + 2 * wave + c;
    }
    return wimg[(size_t)f * 64];
  };

  constexpr int PA = 3, PB = 2;  // prefetch distances (steps) of the A and B windows
  intx4 qa[PA][2];
  intx2 res[2][4][4];  // residual: (output tile c, group g, register quad q), 4 int16
  {
    const int cp = lane & 31, half = lane >> 5;
    const int odd = cp & 1;
    // taps of the channel pair (64 w + 2 cp, + 1) as int16 pairs and the two
    // biases 512 b, from the 96-byte record of its channel quad
    uint32_t wt[9];
    int bias0, bias1;
    {
      const intx4* wsrc = (const intx4*)a.dww + 6 * (16 * wave + (cp >> 1));
      intx4 q0 = wsrc[0], q1 = wsrc[1], q2 = wsrc[2], q3 = wsrc[3], q4 = wsrc[4];
      intx2 q5 = *(const intx2*)(wsrc + 5);
      asm volatile("" : "+v"(q0), "+v"(q1), "+v"(q2), "+v"(q3), "+v"(q4), "+v"(q5));
      int wd[22];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        wd[i] = q0[i];
        wd[4 + i] = q1[i];
        wd[8 + i] = q2[i];
        wd[12 + i] = q3[i];
        wd[16 + i] = q4[i];
      }
      wd[20] = q5[0];
      wd[21] = q5[1];
      // wd[i] for the even lane, wd[j] for the odd one, selected by mask (a
      // conditional index would put wd in scratch memory)
      const uint32_t msk = 0u - (uint32_t)odd;
      auto pick = [&](int i, int j) __attribute__((always_inline)) {
        return (uint32_t)wd[i] ^ (((uint32_t)wd[i] ^ (uint32_t)wd[j]) & msk);
      };
#pragma unroll
      for (int t = 0; t < 9; ++t) wt[t] = pick(2 * t, 2 * t + 1);  // tap t: pair 0 or 1 of the quad
      bias0 = (int)pick(18, 20);  // biases of the quad's channels 0 .. 3 at words 18 .. 21
      bias1 = (int)pick(19, 21);
    }
#pragma unroll
    for (int s = 0; s < PA; ++s)
#pragma unroll
      for (int c = 0; c < 2; ++c) qa[s][c] = afrag(s, c);
    if (wave == 0) {
#pragma unroll
      for (int i = 0; i < 2; ++i) dma16((const char*)a.b1 + i * 1024 + lane * 16, smem + OCORR + i * 1024);
      dma16((const char*)a.b2 + lane * 16, smem + OCORR + 2048);
    }
    char* const band = smem + wave * REG;
    auto band_load = [&](int i) __attribute__((always_inline)) {
      const int S = i * 64 + lane;
      const int bp = S >> 3, u = S & 7;
      const int by = bp / BW, bx = bp - by * BW;
      const int hy = ty0 - 1 + by, hx = tx0 - 1 + bx;
      const bool in = bp < BH * BW && hy >= 0 && hy < a.h && hx >= 0 && hx < a.w;
      dma16(in ? z + (size_t)(hy * a.w + hx) * C + 64 * wave + 8 * (u ^ bswz(bx)) : zpad, band + i * 1024);
    };
    constexpr int BAND_FIRST = 14;
    if (first) {
#pragma unroll
      for (int i = 0; i < BAND_FIRST; ++i) band_load(i);
    }
    int va[TW / 2 + 2];
#pragma unroll
    for (int i = 0; i < TW / 2 + 2; ++i) {
      const int col = half ? TW + 1 - i : i;
      va[i] = col * 128 + (((cp >> 2) ^ bswz(col)) << 4) + (cp & 3) * 4;
    }
    // taps of a row as dot2 pairs (mirrored for half 1): (A0, A1) . (z[k],
    // z[k + 1]) and (0, A2) . (z[k + 1], z[k + 2]) in the lane's column order
    uint32_t W0a[3], W0b[3], W1a[3], W1b[3];
#pragma unroll
    for (int ky = 0; ky < 3; ++ky) {
      const uint32_t l = half ? wt[3 * ky + 2] : wt[3 * ky], m = wt[3 * ky + 1], r = half ? wt[3 * ky] : wt[3 * ky + 2];
      W0a[ky] = __builtin_amdgcn_perm(m, l, 0x05040100u);
      W0b[ky] = r << 16;
      W1a[ky] = __builtin_amdgcn_perm(m, l, 0x07060302u);
      W1b[ky] = r & 0xFFFF0000u;
    }
    // output (row r, step k) of the pair: column x = k (half 0) or 15 - k
    // (half 1); its quad's digits go to a's fragments (group r / 2, k-step
    // 2 w + cp / 16, digit: hi from the even lane, lo from the odd one), lane
    // slot 16 (r % 2) + x + 32 ((cp / 8) % 2), dword (cp / 2) % 4
    int wa[2][TW / 2];
#pragma unroll
    for (int rho = 0; rho < 2; ++rho)
#pragma unroll
      for (int k = 0; k < TW / 2; ++k) {
        const int x = half ? TW - 1 - k : k;
        wa[rho][k] = a_off(0, 2 * (2 * wave + (cp >> 4)) + odd) + bslot(16 * rho + x + 32 * ((cp >> 3) & 1)) * 16 +
                     ((cp >> 1) & 3) * 4;
      }
    // the even lane of a quad takes the high digits of (own pair, partner's),
    // the odd lane the low digits of (partner's, own)
    const uint32_t dsel = odd ? 0x02000604u : 0x07050301u, dxor = odd ? 0x80808080u : 0u;
    uint32_t P0[BH][TW / 2 + 1], P1[BH][TW / 2 + 1];
    auto load_row = [&](int y) __attribute__((always_inline)) {
      uint32_t vr[TW / 2 + 2];
#pragma unroll
      for (int i = 0; i < TW / 2 + 2; ++i) vr[i] = *(const uint32_t*)(band + y * BROW + va[i]);
#pragma unroll
      for (int i = 0; i < TW / 2 + 1; ++i) {
        P0[y][i] = __builtin_amdgcn_perm(vr[i + 1], vr[i], 0x05040100u);
        P1[y][i] = __builtin_amdgcn_perm(vr[i + 1], vr[i], 0x07060302u);
      }
    };
    auto sdot = [](uint32_t w, uint32_t v, int acc) __attribute__((always_inline)) {
      return __builtin_amdgcn_sdot2(__builtin_bit_cast(short2v, w), __builtin_bit_cast(short2v, v), acc, false);
    };
    auto dw_out = [&](int r, int k) __attribute__((always_inline)) {
      int a0 = bias0, a1 = bias1;
#pragma unroll
      for (int ky = 0; ky < 3; ++ky) {
        a0 = sdot(W0a[ky], P0[r + ky][k], a0);
        a0 = sdot(W0b[ky], P0[r + ky][k + 1], a0);
        a1 = sdot(W1a[ky], P1[r + ky][k], a1);
        a1 = sdot(W1b[ky], P1[r + ky][k + 1], a1);
      }
      const uint32_t d = pack_sat(rhe13(a0), rhe13(a1));
      const uint32_t p = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)d, 0xB1, 0xF, 0xF, false);  // lane ^ 1
      *(uint32_t*)(smem + wa[r & 1][k] + 16 * (r >> 1) * XF) = __builtin_amdgcn_perm(p, d, dsel) ^ dxor;
    };
    auto dw_row = [&](int r) __attribute__((always_inline)) {
#pragma unroll
      for (int k = 0; k < TW / 2; ++k) dw_out(r, k);
    };
    // the residual of the wave's outputs is its band's interior: (c, g, q),
    // lane = pixel 32 g + lane % 32 of the tile (band row 1 + 2 g + n / 16,
    // column 1 + n % 16), channels 32 c + 8 q + 4 h .. + 3 of the wave's 64
    auto read_residual = [&]() __attribute__((always_inline)) {
      const int n = lane & 31, x = 1 + (n & 15);
      const char* rb = band + (1 + (n >> 4)) * BROW + x * 128 + 8 * h;
      const int sw = bswz(x);
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int g = 0; g < 4; ++g)
#pragma unroll
          for (int q = 0; q < 4; ++q) res[c][g][q] = *(const intx2*)(rb + 2 * g * BROW + (((4 * c + q) ^ sw) << 4));
    };
    if constexpr (first) {
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
      read_residual();
    } else {
      // pass 1, before this block's ring is known: the outputs that read only
      // the interior (rows 1 .. 6, steps 1 .. 7 of each half row), and the
      // residual
      auto load_inner = [&](int y) __attribute__((always_inline)) {
        uint32_t vr[TW / 2 + 2];
#pragma unroll
        for (int i = 1; i < TW / 2 + 2; ++i) vr[i] = *(const uint32_t*)(band + y * BROW + va[i]);
#pragma unroll
        for (int i = 1; i < TW / 2 + 1; ++i) {
          P0[y][i] = __builtin_amdgcn_perm(vr[i + 1], vr[i], 0x05040100u);
          P1[y][i] = __builtin_amdgcn_perm(vr[i + 1], vr[i], 0x07060302u);
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
      read_residual();
      // the ring, once every neighbouring tile has published block b - 1
      if (wave == 0 && lane < 9 && lane != 4) {
        const int ny = tyi + lane / 3 - 1, nx = txi + lane % 3 - 1;
        if (ny >= 0 && ny < tiles_y && nx >= 0 && nx < tiles_x) {
          const int* f = flags + ny * tiles_x + nx;
          for (int spin = 0; __hip_atomic_load(f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < base + b; ++spin) {
            if (spin > (1 << 16)) {  // about 0.1 s: give up, record it
              __hip_atomic_store(status, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
              break;
            }
            __builtin_amdgcn_s_sleep(1);
          }
        }
      }
      lds_barrier();
      // the ring (52 pixels: rows -1 and 8, columns -1 and 16 of rows 0 .. 7)
      // through registers, with device-coherent loads
      constexpr int RING = 2 * BW + 2 * TH;
      intx4 rv[(RING * 8 + 63) / 64];
      int ro[(RING * 8 + 63) / 64];
#pragma unroll
      for (int i = 0; i < (RING * 8 + 63) / 64; ++i) {
        const int S = i * 64 + lane, r = S >> 3, u = S & 7;
        const int by = r < BW ? 0 : r < 2 * BW ? BH - 1 : 1 + (r - 2 * BW) % TH;
        const int bx = r < BW ? r : r < 2 * BW ? r - BW : (r < 2 * BW + TH ? 0 : BW - 1);
        const int hy = ty0 - 1 + by, hx = tx0 - 1 + bx;
        const bool in = S < RING * 8 && hy >= 0 && hy < a.h && hx >= 0 && hx < a.w;
        rv[i] = load_coherent16i(in ? z + (size_t)(hy * a.w + hx) * C + 64 * wave + 8 * u : zpad);
        ro[i] = S < RING * 8 ? by * BROW + bx * 128 + ((u ^ bswz(bx)) << 4) : -1;
      }
      static_assert((RING * 8 + 63) / 64 == 7, "seven ring loads per lane");
      asm volatile("s_waitcnt vmcnt(0)"
                   : "+v"(rv[0]), "+v"(rv[1]), "+v"(rv[2]), "+v"(rv[3]), "+v"(rv[4]), "+v"(rv[5]), "+v"(rv[6])
                   :
                   : "memory");
#pragma unroll
      for (int i = 0; i < (RING * 8 + 63) / 64; ++i)
        if (ro[i] >= 0) *(intx4*)(band + ro[i]) = rv[i];
      // pass 2: the outputs that read the ring
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
  // the correction loads of wave 0 (the band waits above cover them on a first block)
  if (!first) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  lds_barrier();  // a complete; every wave holds its residual, the bands are free

  // ---- 2, 3. pw1 (steps 0 .. 63) and pw2 (steps 64 .. 127)
  intx16 acc[2][4];  // pw1: chunk c, group g; pw2: output tile c, group g
  auto zero_acc = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int g = 0; g < 4; ++g) acc[c][g] = intx16{};
  };
  auto shift_acc = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int g = 0; g < 4; ++g)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[c][g][i] = (int)((uint32_t)acc[c][g][i] << 8);
  };
  // acc = (acc << 8) + corr, corr of rows row0[c] + drow(i, h) from LDS
  auto shift_corr = [&](int row00, int row01) __attribute__((always_inline)) {
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int* cb = (const int*)(smem + OCORR) + (c ? row01 : row00) + 4 * h;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const intx4 cv = *(const intx4*)(cb + 8 * q);
#pragma unroll
        for (int g = 0; g < 4; ++g)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            acc[c][g][4 * q + e] = (int)(((uint32_t)acc[c][g][4 * q + e] << 8) + (uint32_t)cv[e]);
      }
    }
  };
  // rescale, integer LeakyReLU (slope 819 / 8192) as max(h, RHE(819 h / 2^13)),
  // digits of chunk c of the round to hidden slot 2 w + c: fragments
  // (g, 2 (2 w + c)) (hi) and + 1 (lo), off(g, f) placing fragment (g, f)
  auto leaky_write = [&](auto off) __attribute__((always_inline)) {
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        uint32_t d[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          int v[2];
#pragma unroll
          for (int u = 0; u < 2; ++u) {
            const int hv = rescale13c(acc[c][g][2 * e + u]);
            const int m = 819 * hv;  // |m| < 2^25
            v[u] = max(hv, (m + 4095 + ((m >> 13) & 1)) >> 13);
          }
          d[e] = pack_sat(v[0], v[1]);
        }
        intx4 gh, gl;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          gh[i] = (int)digits_hi(d[2 * i], d[2 * i + 1]);
          gl[i] = (int)digits_lo(d[2 * i], d[2 * i + 1]);
        }
        const int f = 2 * (2 * wave + c);
        *(intx4*)(smem + off(g, f) + myslot) = gh;
        *(intx4*)(smem + off(g, f + 1) + myslot) = gl;
      }
  };
  // B fragment of step t, group g: a (pw1: k-step t % 8, digit pass % 2), then
  // the hidden layer (pw2: chunk (t - 64) % 16, digit pass % 2; chunks 0 .. 7
  // over the bands, 8 .. 15 over a)
  auto bfrag = [&](int t, int g) __attribute__((always_inline)) {
    int off;
    if (t < 64) {
      off = a_off(g, 2 * (t & 7) + ((t >> 3) & 1));
    } else {
      const int u = t - 64, d = (u >> 4) & 1, j = u & 15;
      off = j < 8 ? h0_off(g, 2 * j + d) : a_off(g, 2 * (j - 8) + d);
    }
    return *(const intx4*)(smem + off + myslot);
  };
  zero_acc();
  intx4 qb[PB][4];
#pragma unroll
  for (int s = 0; s < PB; ++s)
#pragma unroll
    for (int g = 0; g < 4; ++g) qb[s][g] = bfrag(s, g);
  __builtin_amdgcn_sched_barrier(0);
  auto step = [&](auto tc) __attribute__((always_inline)) {
    constexpr int t = decltype(tc)::value;
    if constexpr (t == 32) {
      // round 0 done: its hidden layer over the bands (no reader before the
      // hand-off barrier of step 64), then round 1
      leaky_write(h0_off);
      zero_acc();
    }
    if constexpr (t == 64) {
      // round 1 done: once every wave is past its last read of a, its hidden
      // layer replaces a
      lds_barrier();
      leaky_write(a_off);
      zero_acc();
      lds_barrier();
#pragma unroll
      for (int s = 0; s < PB; ++s)
#pragma unroll
        for (int g = 0; g < 4; ++g) qb[s][g] = bfrag(t + s, g);
    }
    // pass boundaries: hh -> hl (shift), lh -> ll (shift and correction)
    if constexpr ((t < 64 && (t & 31) == 8) || t == 64 + 16) shift_acc();
    if constexpr (t < 64 && (t & 31) == 24) shift_corr(32 * (8 * (t >> 5) + 2 * wave), 32 * (8 * (t >> 5) + 2 * wave + 1));
    if constexpr (t == 64 + 48) shift_corr(2 * C + 64 * wave, 2 * C + 64 * wave + 32);
    intx4 A[2], B[4];
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      A[c] = qa[t % PA][c];
      if (t + PA < NT) qa[t % PA][c] = afrag(t + PA, c);
    }
    // the B window restarts after the round-1 hand-off (step 64)
    const bool bnext = t + PB < NT && (t >= 64 || t + PB < 64);
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      B[g] = qb[t % PB][g];
      if (bnext) qb[t % PB][g] = bfrag(t + PB, g);
    }
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int g = 0; g < 4; ++g) acc[c][g] = mfma_i8(A[c], B[g], acc[c][g]);
    __builtin_amdgcn_sched_barrier(0);
  };
  unrolled(step, std::make_integer_sequence<int, NT>{});

  lds_barrier();  // every wave is done reading the hidden layer
  // the block output of (c, g, q): clip(residual + clip(RHE(acc / 8192))),
  // four int16 packed in two dwords (channels 32 c + 8 q + 4 h .. + 3 of the
  // wave's 64, pixel 32 g + lane % 32)
  auto out4 = [&](int c, int g, int q) __attribute__((always_inline)) {
    const intx2 r = res[c][g][q];
    intx2 o;
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      // saturating packed int16 add of the residual pair and the rescaled pair
      // (from inline asm: the vector saturating-add builtin was miscompiled
      // here, adding the first residual word to both pairs)
      const uint32_t v = pack_sat(rhe13(acc[c][g][4 * q + 2 * e]), rhe13(acc[c][g][4 * q + 2 * e + 1]));
      int sum;
      asm("v_pk_add_i16 %0, %1, %2 clamp" : "=v"(sum) : "v"(r[e]), "v"(v));
      o[e] = sum;
    }
    return o;
  };
  if (last) {
    // parked in LDS from offset 0 (row = tile pixel, 8-byte unit u of the row
    // at u ^ (row & 15)), stored as 16-byte vectors
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int p = 32 * g + (lane & 31);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int cc = 64 * wave + 32 * c + 8 * q + 4 * h;
          *(intx2*)(smem + p * 512 + (((cc >> 2) ^ (p & 15)) << 3)) = out4(c, g, q);
        }
      }
    lds_barrier();
    int16_t* dst = (int16_t*)a.dst;
#pragma unroll
    for (int i = 0; i < TH * TW * 32 / 256; ++i) {
      const int idx = i * 256 + threadIdx.x;
      const int px = idx >> 5, k8 = idx & 31;
      const int yy = ty0 + (px >> 4), xx = tx0 + (px & 15);
      if (yy < a.h && xx < a.w) {
        const char* ob = smem + px * 512;
        // units 2 k8 and 2 k8 + 1 are the aligned pair at 2 k8 ^ (px & 14), swapped when px is odd
        const intx4 pv = *(const intx4*)(ob + (((2 * k8) ^ (px & 14)) << 3));
        intx4 o;
        o[0] = (px & 1) ? pv[2] : pv[0];
        o[1] = (px & 1) ? pv[3] : pv[1];
        o[2] = (px & 1) ? pv[0] : pv[2];
        o[3] = (px & 1) ? pv[1] : pv[3];
        __builtin_nontemporal_store(o, (intx4*)(dst + (size_t)(yy * a.w + xx) * C + 8 * k8));
      }
    }
  } else {
    // a block of a chain: the output (zero outside the image, the next
    // depthwise's padding) goes into the interior of the wave's own band
    char* const band = smem + wave * REG;
    const bool full = ty0 + TH <= a.h && tx0 + TW <= a.w;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int p = 32 * g + (lane & 31), py = p >> 4, px = p & 15;
      char* const pb = band + (1 + py) * BROW + (1 + px) * 128 + 8 * h;
      const int sw = bswz(1 + px);
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int q = 0; q < 4; ++q) *(intx2*)(pb + (((4 * c + q) ^ sw) << 4)) = out4(c, g, q);
      if (!full && !(ty0 + py < a.h && tx0 + px < a.w)) {
#pragma unroll
        for (int u = 0; u < 8; ++u) *(intx2*)(pb + ((u ^ sw) << 4)) = intx2{};
      }
    }
    // the tile's 44 edge pixels, the wave's 64 channels, to memory
    int16_t* dst = (int16_t*)a.dst;
    constexpr int EDGE = 2 * TW + 2 * (TH - 2);
#pragma unroll
    for (int i = 0; i < (EDGE * 8 + 63) / 64; ++i) {
      const int S = i * 64 + lane, e = S >> 3, u = S & 7;
      const int e6 = e - 2 * TW, side = e6 >= TH - 2 ? 1 : 0;
      const int py = e < TW ? 0 : e < 2 * TW ? TH - 1 : 1 + e6 - side * (TH - 2);
      const int px = e < TW ? e : e < 2 * TW ? e - TW : side * (TW - 1);
      const int yy = ty0 + py, xx = tx0 + px;
      if (S < EDGE * 8 && yy < a.h && xx < a.w) {
        const intx4 v = *(const intx4*)(band + (1 + py) * BROW + (1 + px) * 128 + ((u ^ bswz(1 + px)) << 4));
        store_coherent16i(dst + (size_t)(yy * a.w + xx) * C + 64 * wave + 8 * u, v);
      }
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    lds_barrier();
    if (threadIdx.x == 0) __hip_atomic_store(flags + tile, base + b + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

template <bool CHAIN>
__device__ __forceinline__ void dci128_body(const BlockArgs* blk, int nb, int* flags, int* status) {
  using namespace dciw;
  __shared__ __attribute__((aligned(1024))) char smem[SMEM];
  const int tiles_x = (blk[0].w + TW - 1) / TW, tiles_y = (blk[0].h + TH - 1) / TH;
  const int tile = xcd_tile(blockIdx.x, gridDim.x);
  if (tile >= tiles_x * tiles_y) return;
  const int wave0 = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if constexpr (!CHAIN) {
    dci128_block<false, true, true>(smem, blk[0], 0, tile, tiles_x, tiles_y, wave0, 0, nullptr, nullptr);
  } else {
    const int base = __builtin_amdgcn_readfirstlane(__hip_atomic_load(flags + tile, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
    dci128_block<true, true, false>(smem, blk[0], 0, tile, tiles_x, tiles_y, wave0, base, flags, status);
    for (int b = 1; b < nb - 1; ++b)
      dci128_block<true, false, false>(smem, blk[b], b, tile, tiles_x, tiles_y, wave0, base, flags, status);
    dci128_block<true, false, true>(smem, blk[nb - 1], nb - 1, tile, tiles_x, tiles_y, wave0, base, flags, status);
  }
}

__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void k_dcblock128_i16(BlockArgs a) {
  dci128_body<false>(&a, 1, nullptr, nullptr);
}

__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void k_dcchain128_i16(DcChainArgs ca) {
  dci128_body<true>(ca.blk, ca.nb, ca.flags, ca.status);
}

hipError_t launch_dcblock128_i16(const BlockArgs& a, hipStream_t st) {
  launch(k_dcblock128_i16, dim3(dc_grid(a.h, a.w)), dim3(256), st, a);
  return hipGetLastError();
}

hipError_t launch_dcchain128_i16(const DcChainArgs& ca, hipStream_t st) {
  if (ca.nb < 2 || ca.nb > kMaxChain) return hipErrorInvalidValue;
  launch(k_dcchain128_i16, dim3(dc_grid(ca.blk[0].h, ca.blk[0].w)), dim3(256), st, ca);
  return hipGetLastError();
}

// Workgroups of the integer chain kernel that fit the device at once.
int dcchain128_i16_resident() {
  int dev = 0, per_cu = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  const hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_dcchain128_i16, 256, 0);
  return e == hipSuccess ? per_cu * cus : 0;
}

}  // namespace nc
