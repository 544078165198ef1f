// C ABI, weight preparation and the per-frame kernel schedule.
//
// The schedule follows the paper's encoding / decoding pipeline (Supp. B.3):
// encoding runs patch embed -> temporal fuse -> encoder blocks -> downsample ->
// prior/quantiser/bits -> decoder (upsample -> fuse -> blocks) and keeps the
// decoder output f_t as the next context without reconstructing the frame;
// decoding runs prior -> decoder -> reconstruction.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <string>
#include <type_traits>
#include <vector>

#include "../../include/ncodec.h"
#include "common.hpp"
#include "internal.hpp"

using namespace nc;

namespace {
thread_local std::string g_create_error;
}

namespace nc {
thread_local LaunchEvents g_launch_events;

ncodec_status set_error(ncodec_status st, const std::string& msg) {
  g_create_error = msg;
  return st;
}
}  // namespace nc

namespace {

constexpr size_t kAlign = 256;
constexpr int kNumQp = 64;  // rate points of the vector banks
size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

bool cfg_valid(const ncodec_config* c, std::string* why) {
  if (!c) { if (why) *why = "cfg is NULL"; return false; }
  if (c->height < 16 || c->width < 16 || c->height > 8192 || c->width > 8192 || c->height % 16 || c->width % 16) {
    if (why) *why = "height and width must be multiples of 16 in [16, 8192]";
    return false;
  }
  if (c->channels != 64 && c->channels != 128 && c->channels != 256 && c->channels != 384 && c->channels != 512) {
    if (why) *why = "channels must be 64, 128, 256, 384 or 512";
    return false;
  }
  if (c->n_enc_blocks < 0 || c->n_enc_blocks > 32 || c->n_dec_blocks < 0 || c->n_dec_blocks > 32) {
    if (why) *why = "block counts must be in [0, 32]";
    return false;
  }
  if (c->path != NCODEC_PATH_FP16 && c->path != NCODEC_PATH_INT16) {
    if (why) *why = "path must be NCODEC_PATH_FP16 or NCODEC_PATH_INT16";
    return false;
  }
  if (c->block != NCODEC_BLOCK_LRELU && c->block != NCODEC_BLOCK_GATED) {
    if (why) *why = "block must be NCODEC_BLOCK_LRELU or NCODEC_BLOCK_GATED";
    return false;
  }
  if (c->n_fe_blocks < 0 || c->n_fe_blocks > 32 || c->n_rg_blocks < 0 || c->n_rg_blocks > 32) {
    if (why) *why = "feature-extractor and reconstruction-generation block counts must be in [0, 32]";
    return false;
  }
  if (c->qp_banks != 0 && c->qp_banks != 1) {
    if (why) *why = "qp_banks must be 0 or 1";
    return false;
  }
  if (c->hyperprior != 0 && c->hyperprior != 1) {
    if (why) *why = "hyperprior must be 0 or 1";
    return false;
  }
  if (c->hyperprior && (c->channels < 128 || c->height % 32 || c->width % 32)) {
    if (why) *why = "the two-step entropy model needs C >= 128 and H, W multiples of 32";
    return false;
  }
  return true;
}

constexpr int kCZ = 64;  // channels of the hyper latent z

size_t hyper_count(int C) {
  return (size_t)kCZ * C * 4 + kCZ + (size_t)8 * C * kCZ + 8 * C + (size_t)C * (C / 2) + C + (size_t)kNumQp * kCZ;
}

size_t weight_count(const ncodec_config& c) {
  const size_t C = (size_t)c.channels;
  const size_t hid = c.block == NCODEC_BLOCK_GATED ? C : 2 * C;  // pw2 input channels
  const size_t blk = C * 9 + C + 2 * C * C + 2 * C + C * hid + C;
  return C * 192 + C + 2 * C * C + C + c.n_enc_blocks * blk + 4 * C * C + C + 2 * C * C + 2 * C + 4 * C * C + 4 * C +
         2 * C * C + C + c.n_dec_blocks * blk + 192 * C + 192 + (size_t)(c.n_fe_blocks + c.n_rg_blocks) * blk +
         (c.qp_banks ? 4 * (size_t)kNumQp * C : 0) + (c.hyperprior ? hyper_count(c.channels) : 0);
}

// fp16(w q) with one rounding: the precision of every weight of the image.
float fold16(float w, double q) { return (float)(f16)((double)w * q); }

// ---------------------------------------------------------------- weight image
struct ConvDev {
  size_t w = 0, wlo = 0, bias = 0;
};
struct BlockDev {
  size_t dww = 0, dwb = 0;
  ConvDev pw1, pw2;
};

struct Image {
  std::vector<uint8_t> bytes;
  size_t add(size_t n) {
    const size_t off = align_up(bytes.size());
    bytes.resize(off + n);
    return off;
  }
  template <class T> T* at(size_t off) { return (T*)(bytes.data() + off); }
};

int16_t q16(float w) {  // round(8192 w) with round-half-even, saturated (Alg. 1)
  double v = std::nearbyint((double)w * 8192.0);
  v = std::fmin(std::fmax(v, -32768.0), 32767.0);
  return (int16_t)v;
}

struct Packer {
  const ncodec_config& cfg;
  Image& img;
  bool is_int;
  std::string* err;
  bool ok = true;

  // Pointwise-type conv, W is N x K row-major (source row stride ldw); row(n') and col(k')
  // give the source indices of packed row n' and packed contraction index k'.
  template <class RowMap, class ColMap>
  ConvDev gemm(const float* W, const float* b, int N, int K, int ldw, RowMap row, ColMap col) {
    ConvDev d;
    if (!is_int) {
      d.w = img.add((size_t)N * K * 2);
      d.bias = img.add((size_t)N * 4);
      f16* wp = img.at<f16>(d.w);
      float* bp = img.at<float>(d.bias);
      const int ks = K / 16;
      for (int mt = 0; mt < N / 32; ++mt)
        for (int s = 0; s < ks; ++s)
          for (int l = 0; l < 64; ++l)
            for (int e = 0; e < 8; ++e) {
              const int n = 32 * mt + (l & 31), k = 16 * s + 8 * (l >> 5) + e;
              wp[(((size_t)mt * ks + s) * 64 + l) * 8 + e] = (f16)W[(size_t)row(n) * ldw + col(k)];
            }
      for (int n = 0; n < N; ++n) bp[n] = (float)(f16)b[row(n)];
      return d;
    }
    d.w = img.add((size_t)N * K);
    d.wlo = img.add((size_t)N * K);
    d.bias = img.add((size_t)N * 4);
    int8_t* hp = img.at<int8_t>(d.w);
    int8_t* lp = img.at<int8_t>(d.wlo);
    int32_t* cp = img.at<int32_t>(d.bias);
    const int ks = K / 32;
    for (int mt = 0; mt < N / 32; ++mt)
      for (int s = 0; s < ks; ++s)
        for (int l = 0; l < 64; ++l)
          for (int e = 0; e < 16; ++e) {
            const int n = 32 * mt + (l & 31), k = 16 * (l >> 5) + 32 * s + e;
            const int wi = q16(W[(size_t)row(n) * ldw + col(k)]);
            if (wi > 32639) {
              if (ok && err) *err = "integer weight above 32639 (|w| >= 3.984) cannot be split into int8 digits";
              ok = false;
            }
            const int lo = ((wi + 128) & 255) - 128;
            const int hi = (wi - lo) / 256;
            const size_t at = (((size_t)mt * ks + s) * 64 + l) * 16 + e;
            hp[at] = (int8_t)hi;
            lp[at] = (int8_t)lo;
          }
    for (int n = 0; n < N; ++n) {
      int64_t sum = 0;
      for (int k = 0; k < K; ++k) sum += q16(W[(size_t)row(n) * ldw + col(k)]);
      const int64_t corr = 512 * (int64_t)q16(b[row(n)]) + 128 * sum;
      cp[n] = (int32_t)(uint32_t)(uint64_t)corr;  // wraps like the int32 accumulator
    }
    return d;
  }

  ConvDev plain(const float* W, const float* b, int N, int K) {
    return gemm(W, b, N, K, K, [](int n) { return n; }, [](int k) { return k; });
  }

  BlockDev block(const float*& cur) {
    const int C = cfg.channels;
    const bool gated = cfg.block == NCODEC_BLOCK_GATED;
    BlockDev d;
    const float* dw = cur; cur += (size_t)C * 9;
    const float* dwb = cur; cur += C;
    const float* w1 = cur; cur += (size_t)2 * C * C;
    const float* b1 = cur; cur += 2 * C;
    const float* w2 = cur; cur += (size_t)C * (gated ? C : 2 * C);
    const float* b2 = cur; cur += C;
    if (!is_int) {
      // fp16: 48 bytes per channel pair (c, c+1): 9 taps as (w_c, w_c+1) fp16
      // pairs, the two biases as fp32, one pad word; the block's depthwise
      // lane for the pair loads it with three 16-byte loads.
      d.dww = img.add((size_t)C / 2 * 48);
      d.dwb = d.dww;
      uint32_t* wp = img.at<uint32_t>(d.dww);
      for (int p = 0; p < C / 2; ++p) {
        uint32_t* q = wp + 12 * p;
        for (int t = 0; t < 9; ++t) {
          const f16 lo = (f16)dw[(2 * p) * 9 + t], hi = (f16)dw[(2 * p + 1) * 9 + t];
          uint16_t ul, uh;
          std::memcpy(&ul, &lo, 2);
          std::memcpy(&uh, &hi, 2);
          q[t] = (uint32_t)ul | ((uint32_t)uh << 16);
        }
        for (int e = 0; e < 2; ++e) {
          const float bv = (float)(f16)dwb[2 * p + e];
          std::memcpy(&q[9 + e], &bv, 4);
        }
        q[11] = 0;
      }
    } else {
      // int16: 96 bytes per channel quad (c .. c+3): for each of the 9 taps the
      // int16 pairs (w_c, w_c+1) and (w_c+2, w_c+3), then the four biases
      // 512 b (int32), two pad words.
      d.dww = img.add((size_t)C / 4 * 96);
      d.dwb = d.dww;
      uint32_t* wp = img.at<uint32_t>(d.dww);
      for (int q = 0; q < C / 4; ++q) {
        uint32_t* o = wp + 24 * q;
        for (int t = 0; t < 9; ++t)
          for (int e = 0; e < 2; ++e) {
            const uint32_t lo = (uint16_t)q16(dw[(4 * q + 2 * e) * 9 + t]);
            const uint32_t hi = (uint16_t)q16(dw[(4 * q + 2 * e + 1) * 9 + t]);
            o[2 * t + e] = lo | (hi << 16);
          }
        for (int e = 0; e < 4; ++e) {
          const int32_t bv = 512 * (int32_t)q16(dwb[4 * q + e]);
          std::memcpy(&o[18 + e], &bv, 4);
        }
        o[22] = o[23] = 0;
      }
    }
    if (C > 256) {
      // wide block (three launches): the pointwise convs as plain GEMM images;
      // gated form: pw1 packed row n' = 64 t + r holds h1 row 32 t + r (r < 32),
      // else h2 row C + 32 t + r - 32, so every 64-row group gates 32 channels
      if (gated)
        d.pw1 = gemm(w1, b1, 2 * C, C, C,
                     [C](int n) { return (n % 64 < 32) ? 32 * (n / 64) + n % 64 : C + 32 * (n / 64) + n % 64 - 32; },
                     [](int k) { return k; });
      else
        d.pw1 = gemm(w1, b1, 2 * C, C, C, [](int n) { return n; }, [](int k) { return k; });
      const int hid = gated ? C : 2 * C;
      d.pw2 = gemm(w2, b2, C, hid, hid, [](int n) { return n; }, [](int k) { return k; });
      return d;
    }
    // Gated form (both paths): entry 2p carries h1 rows 32 p .. +31 (pw1 rows
    // 32 p ..), entry 2p + 1 the matching h2 rows (pw1 rows C + 32 p ..) and
    // the pw2 fragments of gated channels 32 p .. +31; entry 2p's pw2 part is
    // unused (zero).  The LeakyReLU form takes hidden rows 32 j .. in entry j.
    auto row1 = [&](int j) { return gated ? (j & 1 ? C : 0) + 32 * (j >> 1) : 32 * j; };
    auto hid0 = [&](int j) { return gated ? 32 * (j >> 1) : 32 * j; };
    const int ld2 = gated ? C : 2 * C;
    if (!is_int) {
      // Chunk-major image: for each 32-channel hidden chunk j, the KS pw1
      // fragments (rows 32j..32j+31, all C inputs), one bias fragment (the 32
      // biases as fp32 at its start, the rest zero), then the 2*MT pw2
      // fragments that consume that chunk.  The pw2
      // contraction index is permuted inside the chunk so that the pw1
      // accumulator registers are directly the pw2 operand.  One chunk is one
      // contiguous copy into LDS.
      const int KS = C / 16, MT = C / 32, NCH = 2 * C / 32, FR = KS + 1 + 2 * MT;
      d.pw1.w = img.add((size_t)NCH * FR * 1024);
      d.pw1.bias = img.add((size_t)2 * C * 4);
      d.pw2.bias = img.add((size_t)C * 4);
      f16* cp = img.at<f16>(d.pw1.w);
      auto kmap = [](int k) { return 8 * ((k % 8) / 4) + 4 * ((k / 8) % 2) + (k % 4); };  // within 16
      for (int j = 0; j < NCH; ++j)
        for (int f = 0; f < FR; ++f)
          for (int l = 0; l < 64; ++l)
            for (int e = 0; e < 8; ++e) {
              float v;
              if (f < KS) {
                const int n = row1(j) + (l & 31), k = 16 * f + 8 * (l >> 5) + e;
                v = w1[(size_t)n * C + k];
              } else if (f == KS) {
                v = 0.f;  // the bias, written below
              } else if (gated && !(j & 1)) {
                v = 0.f;
              } else {
                const int t = (f - KS - 1) / 2, u = (f - KS - 1) % 2;
                const int n = 32 * t + (l & 31);
                const int hidden = hid0(j) + 16 * u + kmap(8 * (l >> 5) + e);
                v = w2[(size_t)n * ld2 + hidden];
              }
              cp[(((size_t)j * FR + f) * 64 + l) * 8 + e] = (f16)v;
            }
      // fragment KS of chunk j: the 32 pw1 biases of its rows as fp32 (fp16 values),
      // the chain's initial accumulator
      for (int j = 0; j < NCH; ++j) {
        float* fb = (float*)(cp + ((size_t)j * FR + KS) * 64 * 8);
        for (int r = 0; r < 32; ++r) fb[r] = (float)(f16)b1[row1(j) + r];
      }
      float* b1p = img.at<float>(d.pw1.bias);
      float* b2p = img.at<float>(d.pw2.bias);
      for (int n = 0; n < 2 * C; ++n) b1p[n] = (float)(f16)b1[n];
      for (int n = 0; n < C; ++n) b2p[n] = (float)(f16)b2[n];
      return d;
    }
    // Integer chunk-major image: per hidden chunk j, the pw1 hi-digit
    // fragments (KSI k-steps of 32), the pw1 lo-digit fragments, then the pw2
    // hi and lo fragments (one k-step: the chunk's 32 hidden channels, in the
    // order of the pw1 accumulator registers).
    const int KSI = C / 32, MT = C / 32, NCH = 2 * C / 32, FR = 2 * KSI + 2 * MT;
    d.pw1.w = img.add((size_t)NCH * FR * 1024);
    d.pw1.bias = img.add((size_t)2 * C * 4);
    d.pw2.bias = img.add((size_t)C * 4);
    int8_t* cp = img.at<int8_t>(d.pw1.w);
    auto kmap = [](int k) { return 8 * ((k % 16) / 4) + 4 * ((k / 16) % 2) + (k % 4); };  // within 32
    auto digit = [&](int wi, bool hi) {
      if (wi > 32639) {
        if (ok && err) *err = "integer weight above 32639 (|w| >= 3.984) cannot be split into int8 digits";
        ok = false;
      }
      const int lo = ((wi + 128) & 255) - 128;
      return (int8_t)(hi ? (wi - lo) / 256 : lo);
    };
    for (int j = 0; j < NCH; ++j)
      for (int f = 0; f < FR; ++f)
        for (int l = 0; l < 64; ++l)
          for (int e = 0; e < 16; ++e) {
            int wi;
            bool hi;
            if (f < 2 * KSI) {
              const int sstep = f % KSI;
              hi = f < KSI;
              const int n = row1(j) + (l & 31), k = 32 * sstep + 16 * (l >> 5) + e;
              wi = q16(w1[(size_t)n * C + k]);
            } else {
              const int t = (f - 2 * KSI) % MT;
              hi = f < 2 * KSI + MT;
              const int n = 32 * t + (l & 31);
              wi = gated && !(j & 1) ? 0 : q16(w2[(size_t)n * ld2 + hid0(j) + kmap(16 * (l >> 5) + e)]);
            }
            cp[(((size_t)j * FR + f) * 64 + l) * 16 + e] = digit(wi, hi);
          }
    int32_t* c1 = img.at<int32_t>(d.pw1.bias);
    int32_t* c2 = img.at<int32_t>(d.pw2.bias);
    for (int i = 0; i < 2 * C; ++i) {  // in entry order: position 32 j + r is row row1(j) + r
      const int n = row1(i / 32) + i % 32;
      int64_t sum = 0;
      for (int k = 0; k < C; ++k) sum += q16(w1[(size_t)n * C + k]);
      c1[i] = (int32_t)(uint32_t)(uint64_t)(512 * (int64_t)q16(b1[n]) + 128 * sum);
    }
    for (int n = 0; n < C; ++n) {
      int64_t sum = 0;
      for (int k = 0; k < ld2; ++k) sum += q16(w2[(size_t)n * ld2 + k]);
      c2[n] = (int32_t)(uint32_t)(uint64_t)(512 * (int64_t)q16(b2[n]) + 128 * sum);
    }
    return d;
  }
};

struct Layout {
  ConvDev pe, fuse_enc, down, head, up, fuse_dec, rec;
  // fp16 path: patch embed + fuse and upsample + fuse folded into one conv each
  ConvDev enc_in, dec_in;
  std::vector<BlockDev> enc, dec, fe, rg;
  size_t sigma_tab = 0;
  size_t sig8 = 0;     // int path, gated block: compact sigmoid table
  size_t ctxF = 0;     // feature extractor output (the temporal context)
  // entropy coder tables
  size_t c_scales = 0, c_tab = 0, c_ktab = 0;
  size_t image_bytes = 0;
  // state and intermediates (offsets from the workspace base)
  size_t feat[2], yhat[2], ed, zA, zB, y, partials, zpad, spare_bits;
  size_t dwa = 0, hid = 0;  // wide blocks (C > 256): depthwise output, hidden layer
  // chains of C = 256 blocks in one launch: one progress word per tile
  // (zero at creation; every launch adds the same count to all) and a
  // timeout flag
  size_t chain_flags = 0, chain_status = 0;
  // entropy coder: scale indices, symbols, per-stream scratch, lengths,
  // offsets, status words, byte count
  size_t kmap, qtmp, rscratch, rlens, rerrs, rcount;
  size_t mu;  // coded decode: the prior's mu (fp32 or int16, NHWC) between scale indices and symbols
  // two-step entropy model
  ConvDev zana, zsyn, step2;
  size_t zsig = 0;     // sigma of each z channel at the current rate point (fp32)
  size_t zk = 0;       // scale index of every z symbol (uint8, CZ x P32 planar)
  size_t zhat = 0, hp = 0, base = 0;
  int64_t n_z = 0;     // z symbols per frame
  int64_t n_sym, n_streams;
  int n_partials;
  size_t total;
};

// Entropy-coder tables (Fig. 4 "AE" / "AD"): NS = 64 scales sigma_j =
// fp32(0.11 (256 / 0.11)^(j / 63)); for each, symbols q = -R .. R (R =
// ceil(8 sigma_j)) and an escape, probabilities of the Gaussian of scale sigma_j
// quantised to 16-bit frequencies f = 1 + floor(p (2^16 - n)) with the
// remainder added at q = 0.
void build_coder_tables(Image& img, Layout& L, bool is_int, std::string* err) {
  constexpr int NS = kCoderScales;
  float sc[NS];
  for (int j = 0; j < NS; ++j) sc[j] = (float)(0.11 * std::pow(256.0 / 0.11, (double)j / (NS - 1)));
  std::vector<uint16_t> tab(kTabStarts), bkt((size_t)NS * 257);
  for (int j = 0; j < NS; ++j) {
    const int R = std::max((int)std::ceil(8.0 * (double)sc[j]), 32);
    const int n = 2 * R + 2;
    const double sg = (double)sc[j] * std::sqrt(2.0);
    std::vector<int64_t> f(n);
    int64_t sum = 0;
    for (int i = 0; i < n; ++i) {
      double p;
      if (i < n - 1) {
        const double a = std::fabs((double)(i - R));
        p = 0.5 * (std::erfc((a - 0.5) / sg) - std::erfc((a + 0.5) / sg));
      } else {
        p = std::erfc((R + 0.5) / sg);
      }
      f[i] = 1 + (int64_t)std::floor(p * (double)(65536 - n));
      sum += f[i];
    }
    f[R] += 65536 - sum;
    int T = 0, U = 0;
    while (T < n && f[T] == 1) ++T;
    while (U < n && f[n - 1 - U] == 1) ++U;
    tab[4 * j] = (uint16_t)R;
    tab[4 * j + 1] = (uint16_t)(tab.size() - kTabStarts);
    tab[4 * j + 2] = (uint16_t)T;
    tab[4 * j + 3] = (uint16_t)U;
    uint32_t start = 0;
    int b = 0;
    for (int i = 0; i < n; ++i) {
      tab.push_back((uint16_t)start);
      while (b < 256 && std::max<uint32_t>(256u * b, (uint32_t)T) < start + (uint32_t)f[i])
        bkt[(size_t)j * 257 + b++] = (uint16_t)i;
      start += (uint32_t)f[i];
    }
    tab.push_back(0);  // closing start, 2^16 mod 2^16
    bkt[(size_t)j * 257 + 256] = (uint16_t)(n - 1);
  }
  if (tab.size() != (size_t)kTabBuckets) {
    if (err) *err = "coder tables: " + std::to_string(tab.size() - kTabStarts) + " starts, expected " +
                    std::to_string(kCoderStarts);
    return;
  }
  tab.insert(tab.end(), bkt.begin(), bkt.end());
  L.c_scales = img.add(NS * 4);
  std::memcpy(img.at<float>(L.c_scales), sc, NS * 4);
  L.c_tab = img.add(tab.size() * 2);
  std::memcpy(img.at<uint16_t>(L.c_tab), tab.data(), tab.size() * 2);
  if (is_int) {
    // scale index of every int16 s_i: sigma = max(softplus(s_i / 512), 0.11)
    L.c_ktab = img.add(65536);
    uint8_t* kt = img.at<uint8_t>(L.c_ktab);
    for (int i = 0; i < 65536; ++i) {
      const double s = (double)(i - 32768) / 512.0;
      const double sigma = std::fmax(s > 30.0 ? s : std::log1p(std::exp(s)), 0.11);
      int j = 0;
      while (j < NS - 1 && (double)sc[j] < sigma) ++j;
      kt[i] = (uint8_t)j;
    }
  }
}

bool build_layout(const ncodec_config& cfg, const float* w, Image& img, Layout& L, std::string* err, double qp = 0) {
  const int C = cfg.channels;
  const bool is_int = cfg.path == NCODEC_PATH_INT16;
  std::vector<float> zeros;
  if (!w) {
    zeros.assign(weight_count(cfg), 0.f);
    w = zeros.data();
  }
  Packer pk{cfg, img, is_int, err};
  const float* cur = w;
  auto take = [&](size_t n) { const float* p = cur; cur += n; return p; };
  // vector banks (Sec. 4.4): q_e, q_d, q_f, q_r at the end of the list, 64
  // rate points each.  Rate qp in [0, 63] takes (1 - t) row i + t row i+1 with
  // i = min(floor(qp), 62), t = qp - i (in double): the row itself at an
  // integer qp, the linear interpolation of the supplementary rate-adjustment
  // section between two rate points otherwise.
  const size_t nb = (size_t)kNumQp * C;
  const size_t nhyper = cfg.hyperprior ? hyper_count(C) : 0;
  const float* bank = cfg.qp_banks ? w + weight_count(cfg) - nhyper - 4 * nb : nullptr;
  std::vector<double> rows[4];
  if (bank) {
    const int i = std::min((int)std::floor(qp), kNumQp - 2);
    const double t = qp - i;
    for (int b = 0; b < 4; ++b) {
      rows[b].resize(C);
      const float* r0 = bank + b * nb + (size_t)i * C;
      for (int c = 0; c < C; ++c) rows[b][c] = (1.0 - t) * (double)r0[c] + t * (double)r0[C + c];
    }
  }
  auto brow = [&](int b) { return rows[b].data(); };
  std::vector<float> fdown, fdown_b, fup, ffe, ffd, frec;
  // fuse conv with its context columns C .. 2C scaled by q_f
  auto fuse_fold = [&](const float* W, std::vector<float>& out) -> const float* {
    if (!bank) return W;
    out.assign(W, W + (size_t)2 * C * C);
    const double* qf = brow(2);
    for (int n = 0; n < C; ++n)
      for (int c = 0; c < C; ++c) out[(size_t)n * 2 * C + C + c] = fold16(out[(size_t)n * 2 * C + C + c], qf[c]);
    return out.data();
  };
  const float* pe_w = take((size_t)C * 192); const float* pe_b = take(C);
  const float* fe_w = take((size_t)2 * C * C); const float* fe_b = take(C);
  if (is_int) {
    L.pe = pk.plain(pe_w, pe_b, C, 192);
    L.fuse_enc = pk.plain(fuse_fold(fe_w, ffe), fe_b, C, 2 * C);
  } else {
    // fp16 path: the patch embed is linear and feeds the fuse conv alone, so
    // fuse(concat(W_pe u + b_pe, F)) = [W_fe W_pe | W_fc] [u; F] + W_fe b_pe + b_fe
    // (W_fe, W_fc: the fuse's columns on e and on the context F), composed
    // in double and rounded to fp16 once
    const float* fc = fuse_fold(fe_w, ffe);
    const int K = 192 + C;
    std::vector<double> acc(192);
    std::vector<float> m((size_t)C * K), mb(C);
    for (int n = 0; n < C; ++n) {
      std::fill(acc.begin(), acc.end(), 0.0);
      double bb = fe_b[n];
      for (int j = 0; j < C; ++j) {
        const double f = fe_w[(size_t)n * 2 * C + j];
        const float* r = pe_w + (size_t)j * 192;
        for (int k = 0; k < 192; ++k) acc[k] += f * (double)r[k];
        bb += f * (double)pe_b[j];
      }
      for (int k = 0; k < 192; ++k) m[(size_t)n * K + k] = (float)acc[k];
      for (int c = 0; c < C; ++c) m[(size_t)n * K + 192 + c] = fc[(size_t)n * 2 * C + C + c];
      mb[n] = (float)bb;
    }
    L.enc_in = pk.plain(m.data(), mb.data(), C, K);
  }
  for (int k = 0; k < cfg.n_enc_blocks; ++k) L.enc.push_back(pk.block(cur));
  const float* dn_w = take((size_t)4 * C * C); const float* dn_b = take(C);
  if (bank) {  // q_e scales the rows of the downsample (y)
    const double* qe = brow(0);
    fdown.assign(dn_w, dn_w + (size_t)4 * C * C);
    fdown_b.assign(dn_b, dn_b + C);
    for (int o = 0; o < C; ++o) {
      for (size_t k = 0; k < (size_t)4 * C; ++k) fdown[(size_t)o * 4 * C + k] = fold16(fdown[(size_t)o * 4 * C + k], qe[o]);
      fdown_b[o] = fold16(fdown_b[o], qe[o]);
    }
    dn_w = fdown.data();
    dn_b = fdown_b.data();
  }
  // packed k' = (2i + j) * C + c  <-  source column c * 4 + 2i + j
  L.down = pk.gemm(dn_w, dn_b, C, 4 * C, 4 * C, [](int n) { return n; }, [C](int k) { return (k % C) * 4 + k / C; });
  const float* hd_w = take((size_t)2 * C * C); const float* hd_b = take(2 * C);
  // packed row n' = 64 t + r: mu row 32 t + r (r < 32), else s row C + 32 t + r - 32
  L.head = pk.gemm(hd_w, hd_b, 2 * C, C, C,
                   [C](int n) { return (n % 64 < 32) ? 32 * (n / 64) + n % 64 : C + 32 * (n / 64) + n % 64 - 32; },
                   [](int k) { return k; });
  const float* up_w = take((size_t)4 * C * C); const float* up_b = take(4 * C);
  const float* fd_w0 = up_w + (size_t)4 * C * C + 4 * C;  // the fuse conv follows in the list
  if (!is_int) {
    // fp16 path: the upsample (then the x2 shuffle) feeds the fuse conv alone,
    // so at sub-position s of the shuffle the pair is one conv on yhat and F:
    // [W_fd W_up^(s) diag(q_d) | W_fc] [yhat; F] + W_fd b_up^(s) + b_fd, with
    // W_up^(s) the upsample rows 4 c + s (channel c of sub-position s); rows
    // packed s C + n, composed in double and rounded to fp16 once
    const double* qd = bank ? brow(1) : nullptr;
    const float* fc = fuse_fold(fd_w0, ffd);
    const int K = 2 * C;
    std::vector<double> acc(C);
    std::vector<float> m((size_t)4 * C * K), mb(4 * C);
    for (int sp = 0; sp < 4; ++sp)
      for (int n = 0; n < C; ++n) {
        std::fill(acc.begin(), acc.end(), 0.0);
        double bb = fd_w0[(size_t)2 * C * C + n];
        for (int j = 0; j < C; ++j) {
          const double f = fd_w0[(size_t)n * 2 * C + j];
          const float* r = up_w + (size_t)(4 * j + sp) * C;
          for (int k = 0; k < C; ++k) acc[k] += f * (double)r[k];
          bb += f * (double)up_b[4 * j + sp];
        }
        float* row = m.data() + (size_t)(sp * C + n) * K;
        for (int k = 0; k < C; ++k) row[k] = (float)(qd ? acc[k] * qd[k] : acc[k]);
        for (int c = 0; c < C; ++c) row[C + c] = fc[(size_t)n * 2 * C + C + c];
        mb[sp * C + n] = (float)bb;
      }
    L.dec_in = pk.plain(m.data(), mb.data(), 4 * C, K);
  }
  if (bank) {  // q_d scales the columns of the upsample (its input yhat)
    const double* qd = brow(1);
    fup.assign(up_w, up_w + (size_t)4 * C * C);
    for (size_t n = 0; n < (size_t)4 * C; ++n)
      for (int c = 0; c < C; ++c) fup[n * C + c] = fold16(fup[n * C + c], qd[c]);
    up_w = fup.data();
  }
  const float* fd_w = take((size_t)2 * C * C); const float* fd_b = take(C);
  if (is_int) {
    // packed row n' = sp * C + c  <-  source row 4c + sp
    L.up = pk.gemm(up_w, up_b, 4 * C, C, C, [C](int n) { return 4 * (n % C) + n / C; }, [](int k) { return k; });
    L.fuse_dec = pk.plain(fuse_fold(fd_w, ffd), fd_b, C, 2 * C);
  }
  for (int k = 0; k < cfg.n_dec_blocks; ++k) L.dec.push_back(pk.block(cur));
  const float* rc_w = take((size_t)192 * C); const float* rc_b = take(192);
  if (bank) {  // q_r scales the columns of the reconstruction (the generated feature)
    const double* qr = brow(3);
    frec.assign(rc_w, rc_w + (size_t)192 * C);
    for (int n = 0; n < 192; ++n)
      for (int c = 0; c < C; ++c) frec[(size_t)n * C + c] = fold16(frec[(size_t)n * C + c], qr[c]);
    rc_w = frec.data();
  }
  if (is_int) {
    L.rec = pk.plain(rc_w, rc_b, 192, C);
  } else {
    // 256 rows, 192 .. 255 zero: the 256-row pointwise kernel computes whole
    // 64-row slices per wave and stores only the 192 frame rows
    std::vector<float> wpad((size_t)256 * C, 0.f), bpad(256, 0.f);
    std::copy(rc_w, rc_w + (size_t)192 * C, wpad.begin());
    std::copy(rc_b, rc_b + 192, bpad.begin());
    L.rec = pk.plain(wpad.data(), bpad.data(), 256, C);
  }
  for (int k = 0; k < cfg.n_fe_blocks; ++k) L.fe.push_back(pk.block(cur));
  for (int k = 0; k < cfg.n_rg_blocks; ++k) L.rg.push_back(pk.block(cur));
  if (bank) cur += 4 * nb;
  if (cfg.hyperprior) {
    // hyper-analysis: like the downsample, packed k' = (2i + j) C + c <- source column 4c + 2i + j
    const float* za_w = take((size_t)kCZ * 4 * C); const float* za_b = take(kCZ);
    L.zana = pk.gemm(za_w, za_b, kCZ, 4 * C, 4 * C, [](int n) { return n; }, [C](int k) { return (k % C) * 4 + k / C; });
    // hyper-synthesis: like the upsample over 2C channels, packed row n' = sp 2C + m <- source row 4m + sp
    const float* zs_w = take((size_t)8 * C * kCZ); const float* zs_b = take(8 * C);
    L.zsyn = pk.gemm(zs_w, zs_b, 8 * C, kCZ, kCZ, [C](int n) { return 4 * (n % (2 * C)) + n / (2 * C); },
                     [](int k) { return k; });
    // second step: like the prior head over C / 2 channels, packed row n' = 64 t + r:
    // dmu row 32 t + r (r < 32), else ds row C/2 + 32 t + r - 32
    const float* s2_w = take((size_t)C * (C / 2)); const float* s2_b = take(C);
    L.step2 = pk.gemm(s2_w, s2_b, C, C / 2, C / 2,
                      [C](int n) { return (n % 64 < 32) ? 32 * (n / 64) + n % 64 : C / 2 + 32 * (n / 64) + n % 64 - 32; },
                      [](int k) { return k; });
    // the z bank row of the rate point (the nearest learned point), sigma floored at 0.11
    const float* zbank = take((size_t)kNumQp * kCZ);
    const int row = std::min((int)std::floor(qp + 0.5), kNumQp - 1);
    L.zsig = img.add(kCZ * 4);
    float* zs = img.at<float>(L.zsig);
    double zsd[kCZ];
    for (int c = 0; c < kCZ; ++c) {
      zsd[c] = std::fmax((double)zbank[(size_t)row * kCZ + c], 0.11);
      zs[c] = (float)zsd[c];
    }
    // scale index of every z symbol (the smallest coder scale >= sigma_z, in double)
    const size_t P32 = (size_t)(cfg.height / 32) * (cfg.width / 32);
    L.zk = img.add(kCZ * P32);
    uint8_t* zk = img.at<uint8_t>(L.zk);
    for (int c = 0; c < kCZ; ++c) {
      int j = 0;
      while (j < kCoderScales - 1 && (double)(float)(0.11 * std::pow(256.0 / 0.11, (double)j / (kCoderScales - 1))) < zsd[c]) ++j;
      std::memset(zk + (size_t)c * P32, j, P32);
    }
  }
  if ((size_t)(cur - w) != weight_count(cfg)) {
    if (err) *err = "internal: parameter walk mismatch";
    return false;
  }
  if (is_int && cfg.block == NCODEC_BLOCK_GATED) {
    // S[v] = RHE(512 sigmoid(4 v / 512)) for every int16 v (the WSiLU's
    // sigmoid, K1-scaled in and out; no entry lies within 1e-6 of a rounding
    // tie).  The kernel reads it from a compact form: s8[a] = S[a] - 256 for
    // 0 <= a < 888, S[a] = 512 above, S[-a] = 512 - S[a].  That form is
    // checked against the full table here.
    constexpr int kSat = 888, kBytes = 896;
    auto S = [](int v) { return (int)std::nearbyint(512.0 / (1.0 + std::exp(-4.0 * (double)v / 512.0))); };
    L.sig8 = img.add(kBytes);
    uint8_t* s8 = img.at<uint8_t>(L.sig8);
    bool shape_ok = S(-32768) == 0;
    for (int a = 0; a < 32768; ++a) {
      const int sa = S(a);
      if (a < kSat) {
        shape_ok = shape_ok && sa >= 256 && sa <= 511;
        s8[a] = (uint8_t)(sa - 256);
      } else {
        shape_ok = shape_ok && sa == 512;
      }
      shape_ok = shape_ok && S(-a) == 512 - sa;
    }
    if (!shape_ok) {
      if (err) *err = "internal: sigmoid table does not have the compact form";
      return false;
    }
  }
  if (is_int) {
    L.sigma_tab = img.add(65536 * 4);
    float* tab = img.at<float>(L.sigma_tab);
    for (int i = 0; i < 65536; ++i) {
      const double s = (double)(i - 32768) / 512.0;
      const double sp = s > 30.0 ? s : std::log1p(std::exp(s));
      tab[i] = (float)std::fmax(sp, 0.11);
    }
  }
  std::string terr;
  build_coder_tables(img, L, is_int, &terr);
  if (!terr.empty()) {
    if (err) *err = "internal: " + terr;
    return false;
  }
  L.image_bytes = align_up(img.bytes.size());

  const size_t P8 = (size_t)(cfg.height / 8) * (cfg.width / 8);
  const size_t P16 = P8 / 4;
  const size_t fb = P8 * C * 2, lb = P16 * C * 2;
  size_t off = L.image_bytes;
  auto alloc = [&](size_t n) { const size_t o = off; off = align_up(off + n); return o; };
  L.feat[0] = alloc(fb); L.feat[1] = alloc(fb);
  L.yhat[0] = alloc(lb); L.yhat[1] = alloc(lb);
  L.ed = alloc(fb); L.zA = alloc(fb); L.zB = alloc(fb);
  if (cfg.n_fe_blocks > 0) L.ctxF = alloc(fb);
  if (C > 256) {  // wide blocks: the depthwise output and the hidden layer
    L.dwa = alloc(fb);
    L.hid = alloc(2 * fb);
  }
  L.y = alloc(lb);
  if (C == 256) {
    const size_t tiles = (size_t)((cfg.height / 8 + 7) / 8) * ((cfg.width / 8 + 15) / 16);
    L.chain_flags = alloc(tiles * 4);
    L.chain_status = alloc(4);
  }
  const size_t P32 = P16 / 4;
  // rate partial sums: the prior's (tiles x passes); with the two-step model
  // also the z quantiser's (one per tile) and the second step's
  int np = is_int ? prior_partials_i16(C, (int)P16) : prior_partials_f16(C, (int)P16);
  if (cfg.hyperprior) np += (int)((P32 + 127) / 128) + (int)((P16 + 127) / 128) * (C / 64);
  L.n_partials = np > kBitsBlocks ? np : kBitsBlocks;
  L.partials = alloc((size_t)L.n_partials * 8);
  L.zpad = alloc((size_t)C * 2);  // zeroed at create and never written
  L.spare_bits = alloc(8);        // bit total of graph replays called without d_bits
  L.n_z = cfg.hyperprior ? (int64_t)P32 * kCZ : 0;
  L.n_sym = (int64_t)P16 * C;
  L.n_streams = (L.n_sym + kRansStream - 1) / kRansStream;
  L.kmap = alloc((size_t)L.n_sym);
  L.qtmp = alloc((size_t)(L.n_sym + L.n_z) * 2);
  L.rscratch = alloc((size_t)L.n_streams * kRansMaxWords * 2);
  L.rlens = alloc((size_t)L.n_streams * 4);
  L.rerrs = alloc((size_t)L.n_streams * 4);
  L.rcount = alloc(4);  // decoder ticket counter: zeroed at create, left at zero by every decode
  L.mu = alloc(P16 * C * 4);
  if (cfg.hyperprior) {
    L.zhat = alloc(P32 * kCZ * 2);
    L.hp = alloc(P16 * 2 * C * 2);
    L.base = alloc(P16 * C * 4);
  }
  L.total = off;
  return pk.ok;
}

}  // namespace

struct ncodec_ctx {
  ncodec_config cfg;
  std::vector<float> host_w;  // canonical weights, kept to refold the vector banks (qp_banks only)
  double qp = 0;  // rate point of the folded banks
  int device;
  hipStream_t stream;
  char* ws;
  Layout L;
  int cur = 0;
  std::string err;
  struct TimedLaunch {
    const char* kind;
    hipEvent_t start, stop;
    int n;  // launches in the interval (a run of consecutive launches of one kind)
  };
  bool timing = false;
  std::vector<TimedLaunch> log;
  // Graph replay: one captured graph per (encode / decode, state parity), with
  // the kernel nodes that touch caller buffers, updated when those change.
  struct CapturedNode {
    const char* kind;
    hipGraphNode_t node;
  };
  struct GraphSlot {
    hipGraph_t graph = nullptr;
    hipGraphExec_t exec = nullptr;
    std::vector<CapturedNode> nodes;
    const void* ptr[3] = {nullptr, nullptr, nullptr};
  };
  bool use_graphs = false;
  GraphSlot graphs[2][2];  // [decode][cur]
  // consecutive C = 256 blocks as one chain launch (when every tile fits
  // the device at once; chain_fit: -1 not yet checked, 0 no, 1 yes)
  bool chains = true;
  int chain_fit = -1;
  // Parallel coding (Fig. 6; supplementary "Parallel Coding"): the coded
  // calls run the entropy coder (encode) or the feature extractor (decode) on
  // a second stream of default priority, joined by events before the call's
  // last launch on the context's stream.
  bool overlap = false;
  hipStream_t aux = nullptr;
  hipEvent_t ev_fork = nullptr, ev_join = nullptr;
  hipStream_t cap_stream = nullptr;
  std::vector<CapturedNode>* capturing = nullptr;
  bool is_int() const { return cfg.path == NCODEC_PATH_INT16; }
  template <class T = void> T* p(size_t off) const { return (T*)(ws + off); }
};

namespace {

ncodec_status fail(ncodec_ctx* ctx, ncodec_status st, const std::string& msg) {
  if (ctx) ctx->err = msg; else g_create_error = msg;
  return st;
}

ncodec_status hip_fail(ncodec_ctx* ctx, hipError_t e, const char* where) {
  return fail(ctx, NCODEC_EHIP, std::string(where) + ": " + hipGetErrorString(e));
}

#define NC_HIP(ctx, expr, where)                          \
  do {                                                    \
    hipError_t _e = (expr);                               \
    if (_e != hipSuccess) return hip_fail(ctx, _e, where); \
  } while (0)

// Runs one launch.  In timing mode the launch's kernel dispatch carries a
// start / stop event pair (hipExtLaunchKernelGGL), so the recorded interval
// is that kernel's execution, without the dispatch gap before it.
template <class F>
hipError_t timed(ncodec_ctx* ctx, const char* kind, F&& launch_fn, int count = 1) {
  if (ctx->capturing) {
    hipError_t e = launch_fn();
    if (e != hipSuccess) return e;
    hipStreamCaptureStatus cs;
    const hipGraphNode_t* deps = nullptr;
    size_t nd = 0;
    e = hipStreamGetCaptureInfo_v2(ctx->stream, &cs, nullptr, nullptr, &deps, &nd);
    if (e == hipSuccess && nd == 1) ctx->capturing->push_back({kind, deps[0]});
    return e;
  }
  if (!ctx->timing) return launch_fn();
  // A run of consecutive launches of one kind (the DC blocks of a transform)
  // shares one interval: the start event of its first launch and the stop
  // event of its last, so the per-launch average includes the gaps between
  // those launches but only one pair of event packets.
  if (!ctx->log.empty() && !std::strcmp(ctx->log.back().kind, kind)) {
    ncodec_ctx::TimedLaunch& t = ctx->log.back();
    hipEvent_t stop = nullptr;
    hipError_t e = hipEventCreate(&stop);
    if (e != hipSuccess) return e;
    g_launch_events = {nullptr, stop};
    e = launch_fn();
    g_launch_events = {};
    if (t.stop) (void)hipEventDestroy(t.stop);
    t.stop = stop;
    t.n += count;
    return e;
  }
  ncodec_ctx::TimedLaunch t{kind, nullptr, nullptr, count};
  hipError_t e = hipEventCreate(&t.start);
  if (e == hipSuccess) e = hipEventCreate(&t.stop);
  if (e == hipSuccess) {
    g_launch_events = {t.start, t.stop};
    e = launch_fn();
    g_launch_events = {};
  }
  ctx->log.push_back(t);
  return e;
}

ncodec_status enter(ncodec_ctx* ctx) {
  if (!ctx) return fail(nullptr, NCODEC_EINVAL, "ctx is NULL");
  hipError_t e = hipSetDevice(ctx->device);
  if (e != hipSuccess) return hip_fail(ctx, e, "hipSetDevice");
  e = hipGetLastError();  // surfaces an earlier asynchronous failure
  if (e != hipSuccess) return hip_fail(ctx, e, "earlier launch");
  return NCODEC_OK;
}

hipError_t pw(ncodec_ctx* ctx, const char* kind, int loader, int epi, const PwArgs& a) {
  return timed(ctx, kind, [&] {
    return ctx->is_int() ? launch_pw_i16(loader, epi, a, ctx->stream) : launch_pw_f16(loader, epi, a, ctx->stream);
  });
}

hipError_t dcblock(ncodec_ctx* ctx, BlockArgs ba) {
  const int C = ctx->cfg.channels;
  const bool gated = ctx->cfg.block == NCODEC_BLOCK_GATED;
  if (gated && ctx->is_int()) ba.sig8 = ctx->p(ctx->L.sig8);
  return timed(ctx, "dcblock", [&] {
    if (ctx->is_int())
      return C == 256 && !gated ? launch_dcblock128_i16(ba, ctx->stream) : launch_dcblock_i16(C, gated, ba, ctx->stream);
    return launch_dcblock_f16(C, gated, ba, ctx->stream);
  });
}

hipError_t prior(ncodec_ctx* ctx, const PriorArgs& pa, int* np) {
  return timed(ctx, "prior", [&] {
    return ctx->is_int() ? launch_prior_i16(pa, ctx->stream, np) : launch_prior_f16(pa, ctx->stream, np);
  });
}

PwArgs conv_args(const ncodec_ctx* ctx, const ConvDev& c, int K, int N, int P) {
  PwArgs a;
  std::memset(&a, 0, sizeof(a));
  a.wfrag = ctx->p(c.w);
  a.wfrag_lo = ctx->is_int() ? ctx->p(c.wlo) : nullptr;
  a.bias = ctx->p(c.bias);
  a.K = K;
  a.N = N;
  a.P = P;
  a.w8 = ctx->cfg.width / 8;
  a.H = ctx->cfg.height;
  a.W = ctx->cfg.width;
  return a;
}

// Whether runs of DC blocks go as chain launches: C = 256 (fp16 either form,
// int the LeakyReLU form), enabled, and every tile of the grid resident on the
// device at once (checked once per context).
bool chains_usable(ncodec_ctx* ctx) {
  const bool gated = ctx->cfg.block == NCODEC_BLOCK_GATED;
  if (!ctx->chains || ctx->cfg.channels != 256 || (ctx->is_int() && gated)) return false;
  if (ctx->chain_fit < 0) {
    const int resident = ctx->is_int() ? dcchain128_i16_resident() : dcchain128_resident(gated);
    ctx->chain_fit = resident >= dc_grid(ctx->cfg.height / 8, ctx->cfg.width / 8) ? 1 : 0;
  }
  return ctx->chain_fit == 1;
}

// One DC block of either form, src -> dst.
hipError_t run_block(ncodec_ctx* ctx, const BlockDev& b, const void* src, void* dst) {
  const int h8 = ctx->cfg.height / 8, w8 = ctx->cfg.width / 8;
  const int C = ctx->cfg.channels;
  if (C > 256) {
    // wide block: depthwise, pw C -> 2C + LeakyReLU (gated: + WSiLU gate), pw
    // 2C (gated: C) -> C + residual
    const Layout& L = ctx->L;
    hipError_t e = timed(ctx, "dcblock_dw", [&] {
      return ctx->is_int() ? launch_dw3x3_i16(src, ctx->p(b.dww), ctx->p(L.dwa), C, h8, w8, ctx->stream)
                           : launch_dw3x3_f16(src, ctx->p(b.dww), ctx->p(L.dwa), C, h8, w8, ctx->stream);
    });
    if (e != hipSuccess) return e;
    PwArgs a = conv_args(ctx, b.pw1, C, 2 * C, h8 * w8);
    a.src0 = ctx->p(L.dwa);
    a.C0 = C;
    const bool gated = ctx->cfg.block == NCODEC_BLOCK_GATED;
    const int hid = gated ? C : 2 * C;  // hidden channels after the activation
    a.dst = ctx->p(L.hid);
    a.Cdst = hid;
    if (gated && ctx->is_int()) a.sig8 = ctx->p<uint8_t>(L.sig8);
    e = pw(ctx, "dcblock_pw1", LD_NHWC, gated ? EP_GATE : EP_LRELU, a);
    if (e != hipSuccess) return e;
    a = conv_args(ctx, b.pw2, hid, C, h8 * w8);
    a.src0 = ctx->p(L.hid);
    a.C0 = hid;
    a.res = src;
    a.dst = dst;
    a.Cdst = C;
    return pw(ctx, "dcblock_pw2", LD_NHWC, EP_RESID, a);
  }
  BlockArgs ba{ctx->p(b.pw1.w), ctx->is_int() ? ctx->p(b.pw1.wlo) : nullptr, ctx->p(b.pw1.bias),
               ctx->p(b.pw2.w), ctx->is_int() ? ctx->p(b.pw2.wlo) : nullptr, ctx->p(b.pw2.bias),
               ctx->p(b.dww), ctx->p(b.dwb), src, dst, h8, w8, ctx->p(ctx->L.zpad)};
  return dcblock(ctx, ba);
}

// Blocks 0 .. n - 1 of `blocks`, block k from src[k] into dst[k] (src[k + 1]
// = dst[k]).  At C = 256 (int path: LeakyReLU form) runs of up to kMaxChain blocks go
// as one chain launch when every tile of the grid fits the device at once;
// otherwise (and for a run of one) one launch per block.  The timing log
// counts blocks either way.
// With down set (the encoder's blocks, fp16) and the run's last launch a
// chain, that launch also runs the 2x2 stride-2 downsample on each tile's last
// block output (into down_y; dst[n - 1] is then not written) and *down_done
// is set; otherwise the caller runs the downsample.
hipError_t run_blocks(ncodec_ctx* ctx, const std::vector<BlockDev>& blocks, const std::vector<const void*>& src,
                      const std::vector<void*>& dst, const ConvDev* down = nullptr, void* down_y = nullptr,
                      bool* down_done = nullptr) {
  const int n = (int)blocks.size();
  const int h8 = ctx->cfg.height / 8, w8 = ctx->cfg.width / 8;
  const bool gated = ctx->cfg.block == NCODEC_BLOCK_GATED;
  const bool chain = n >= 2 && chains_usable(ctx);
  for (int k0 = 0; k0 < n;) {
    const int m = chain ? std::min(n - k0, kMaxChain) : 1;
    if (m == 1) {
      const hipError_t e = run_block(ctx, blocks[k0], src[k0], dst[k0]);
      if (e != hipSuccess) return e;
      ++k0;
      continue;
    }
    DcChainArgs ca;
    std::memset(&ca, 0, sizeof(ca));
    for (int j = 0; j < m; ++j) {
      const BlockDev& b = blocks[k0 + j];
      ca.blk[j] = BlockArgs{ctx->p(b.pw1.w), nullptr, ctx->p(b.pw1.bias), ctx->is_int() ? nullptr : ctx->p(b.pw2.w),
                            nullptr, ctx->p(b.pw2.bias), ctx->p(b.dww), ctx->p(b.dwb), src[k0 + j], dst[k0 + j],
                            h8, w8, ctx->p(ctx->L.zpad)};
    }
    ca.nb = m;
    ca.flags = ctx->p<int>(ctx->L.chain_flags);
    ca.status = ctx->p<int>(ctx->L.chain_status);
    const bool fuse = down && !ctx->is_int() && k0 + m == n;
    if (fuse) {
      ca.down_w = ctx->p(down->w);
      ca.down_b = ctx->p(down->bias);
      ca.down_y = down_y;
      *down_done = true;
    }
    const hipError_t e = timed(ctx, fuse ? "dcblock_down" : "dcblock", [&] {
      return ctx->is_int() ? launch_dcchain128_i16(ca, ctx->stream) : launch_dcchain128_f16(gated, ca, ctx->stream);
    }, m);
    if (e != hipSuccess) return e;
    k0 += m;
  }
  return hipSuccess;
}

// A chain of DC blocks from src, ping-ponging through zA / zB, the last one
// writing `last`; returns the buffer that holds the result (src if empty).
// src and last must not be zA or zB.
hipError_t run_chain(ncodec_ctx* ctx, const std::vector<BlockDev>& blocks, const void* src, void* last,
                     const void** result) {
  std::vector<const void*> srcs;
  std::vector<void*> dsts;
  const void* z = src;
  for (size_t k = 0; k < blocks.size(); ++k) {
    void* dst = k + 1 == blocks.size() ? last : (z == ctx->p(ctx->L.zA) ? ctx->p(ctx->L.zB) : ctx->p(ctx->L.zA));
    srcs.push_back(z);
    dsts.push_back(dst);
    z = dst;
  }
  const hipError_t e = run_blocks(ctx, blocks, srcs, dsts);
  if (e != hipSuccess) return e;
  *result = z;
  return hipSuccess;
}

// The temporal context of this frame: the feature extractor's blocks on
// f_{t-1} into ctxF, or f_{t-1} itself without a feature extractor.
hipError_t temporal_context(ncodec_ctx* ctx, const void** out) {
  const void* f_prev = ctx->p(ctx->L.feat[ctx->cur]);
  if (ctx->L.fe.empty()) {
    *out = f_prev;
    return hipSuccess;
  }
  return run_chain(ctx, ctx->L.fe, f_prev, ctx->p(ctx->L.ctxF), out);
}

// Runs the decoder-side transform from yhat_new (already written) into feat[nxt].
// In an encode with d_bits, the upsample also sums the frame's n_parts rate
// partials into d_bits.
ncodec_status run_decoder(ncodec_ctx* ctx, int nxt, double* d_bits = nullptr, int n_parts = 0) {
  const ncodec_config& c = ctx->cfg;
  const int C = c.channels;
  const int h8 = c.height / 8, w8 = c.width / 8;
  const int P8 = h8 * w8, P16 = P8 / 4;
  const Layout& L = ctx->L;
  const void* f_prev = L.fe.empty() ? ctx->p(L.feat[1 - nxt]) : ctx->p(L.ctxF);  // the temporal context
  void* f_new = ctx->p(L.feat[nxt]);

  void* z = c.n_dec_blocks == 0 ? f_new : ctx->p(L.zA);
  PwArgs a;
  if (ctx->is_int()) {
    a = conv_args(ctx, L.up, C, 4 * C, P16);
    a.src0 = ctx->p(L.yhat[nxt]);
    a.C0 = C;
    a.dst = ctx->p(L.ed);
    a.Cdst = C;
    a.bits_out = d_bits;
    a.sum_base = ctx->p<double>(L.partials);
    a.n_sum = n_parts;
    NC_HIP(ctx, pw(ctx, "up", LD_NHWC, EP_UP, a), "upsample");

    a = conv_args(ctx, L.fuse_dec, 2 * C, C, P8);
    a.src0 = ctx->p(L.ed);
    a.C0 = C;
    a.src1 = f_prev;
    a.C1 = C;
    a.dst = z;
    a.Cdst = C;
    NC_HIP(ctx, pw(ctx, "fuse", LD_NHWC, EP_NHWC, a), "fuse_dec");
  } else {
    // upsample, shuffle and fuse as one conv per sub-position on [yhat; F]
    // (weights composed at load), written through the x2 shuffle
    a = conv_args(ctx, L.dec_in, 2 * C, 4 * C, P16);
    a.src0 = ctx->p(L.yhat[nxt]);
    a.C0 = C;
    a.src1 = f_prev;
    a.C1 = C;
    a.dst = z;
    a.Cdst = C;
    a.bits_out = d_bits;
    a.sum_base = ctx->p<double>(L.partials);
    a.n_sum = n_parts;
    NC_HIP(ctx, pw(ctx, "up_fuse", LD_UP_CTX, EP_UP, a), "upsample + fuse_dec");
  }

  {
    std::vector<const void*> srcs;
    std::vector<void*> dsts;
    for (int k = 0; k < c.n_dec_blocks; ++k) {
      void* dst = (k == c.n_dec_blocks - 1) ? f_new : (z == ctx->p(L.zA) ? ctx->p(L.zB) : ctx->p(L.zA));
      srcs.push_back(z);
      dsts.push_back(dst);
      z = dst;
    }
    NC_HIP(ctx, run_blocks(ctx, L.dec, srcs, dsts), "decoder blocks");
  }
  return NCODEC_OK;
}

// ---- two-step entropy model with the hyper latent z (Sec. 4.4; supplementary
// "Entropy model", "Parallel Coding")
int P16_of(const ncodec_ctx* ctx) { return (ctx->cfg.height / 16) * (ctx->cfg.width / 16); }
// rate partials of a prior launch over P latent pixels with N head rows: one
// per (128-pixel tile, 64-row pass)
int prior_parts(int P, int N) { return ((P + 127) / 128) * (N / 64); }
int P32_of(const ncodec_ctx* ctx) { return (ctx->cfg.height / 32) * (ctx->cfg.width / 32); }

// z = conv2x2/s2(y), quantised: symbols to qz (planar), zhat (NHWC), one rate
// partial per 1/32 tile from *parts on.
hipError_t z_encode(ncodec_ctx* ctx, int16_t* qz, double* parts, int* np) {
  const Layout& L = ctx->L;
  const int C = ctx->cfg.channels;
  PwArgs a = conv_args(ctx, L.zana, 4 * C, kCZ, P32_of(ctx));
  a.src0 = ctx->p(L.y);
  a.Csrc = C;
  a.w8 = ctx->cfg.width / 16;  // the gather reads the 1/16 grid
  a.dst = ctx->p(L.zhat);
  a.Cdst = kCZ;
  a.q_out = qz;
  a.partials = parts;
  a.zsigma = ctx->p<float>(L.zsig);
  return timed(ctx, "zquant", [&] {
    return ctx->is_int() ? launch_zquant_i16(a, ctx->stream, np) : launch_zquant_f16(a, ctx->stream, np);
  });
}

// zhat from the decoded z symbols (fp16: q_z; int: clip(512 q_z)).
hipError_t z_from_symbols(ncodec_ctx* ctx, const int16_t* qz) {
  return timed(ctx, "zhat", [&] {
    return launch_yhat_from_q(qz, nullptr, ctx->p(ctx->L.zhat), kCZ, P32_of(ctx), ctx->is_int(), ctx->stream, kCZ, 0);
  });
}

// hyper parameters [mu_h ; s_h] (NHWC, 2C channels at 1/16) = shuffle2(W_zs zhat + b).
hipError_t hyper_synth(ncodec_ctx* ctx) {
  const Layout& L = ctx->L;
  const int C = ctx->cfg.channels;
  PwArgs a = conv_args(ctx, L.zsyn, kCZ, 8 * C, P32_of(ctx));
  a.src0 = ctx->p(L.zhat);
  a.C0 = kCZ;
  a.dst = ctx->p(L.hp);
  a.Cdst = 2 * C;
  a.w8 = ctx->cfg.width / 16;  // the shuffle writes the 1/16 grid
  return pw(ctx, "hyper", LD_NHWC, EP_UP, a);
}

// Step 1 of the two-step model on a prior call: the hyper parameters are
// added to (mu, s); the second half of the channels leaves (mu, s) in base.
void step1_fields(const ncodec_ctx* ctx, PriorArgs& pa) {
  const int C = ctx->cfg.channels;
  pa.add = ctx->p(ctx->L.hp);
  pa.add_ld = 2 * C;
  pa.add_s = C;
  pa.add_c0 = 0;
  pa.add_f32 = 0;
  pa.split = C / 2;
  pa.base = ctx->p(ctx->L.base);
}

// Step 2: the second-step head on yhat^1 (the first C / 2 channels of
// yhat_t), plus the first step's (mu, s) of the second half, for channels
// C / 2 .. C.
PriorArgs step2_args(const ncodec_ctx* ctx, int nxt, int decode) {
  const int C = ctx->cfg.channels;
  const Layout& L = ctx->L;
  PriorArgs pa;
  std::memset(&pa, 0, sizeof(pa));
  pa.wfrag = ctx->p(L.step2.w);
  pa.wfrag_lo = ctx->is_int() ? ctx->p(L.step2.wlo) : nullptr;
  pa.bias = ctx->p(L.step2.bias);
  pa.K = C / 2;
  pa.N = C;
  pa.yhat_prev = ctx->p(L.yhat[nxt]);
  pa.ld0 = C;
  pa.yhat_new = ctx->p(L.yhat[nxt]);
  pa.sigma_tab = ctx->is_int() ? ctx->p<float>(L.sigma_tab) : nullptr;
  pa.scales = ctx->p<float>(L.c_scales);
  pa.k_tab = ctx->is_int() ? ctx->p<uint8_t>(L.c_ktab) : nullptr;
  pa.C = C;
  pa.P = P16_of(ctx);
  pa.decode = decode;
  pa.c_off = C / 2;
  pa.add = ctx->p(L.base);
  pa.add_ld = C;
  pa.add_s = C / 2;
  pa.add_c0 = C / 2;
  pa.add_f32 = ctx->is_int() ? 0 : 1;
  return pa;
}

// Enqueues one encode on ctx->stream (or records it under capture).
// after_prior (optional) runs once q and the scale indices are enqueued,
// before the decoder part.
template <class Hook = std::nullptr_t>
ncodec_status enqueue_encode(ncodec_ctx* ctx, const void* d_frame, int16_t* d_q, double* d_bits,
                             uint8_t* d_k = nullptr, Hook after_prior = nullptr) {
  ncodec_status st;
  const ncodec_config& c = ctx->cfg;
  const int C = c.channels;
  const int h8 = c.height / 8, w8 = c.width / 8;
  const int P8 = h8 * w8, P16 = P8 / 4;
  const Layout& L = ctx->L;
  const int cur = ctx->cur, nxt = 1 - cur;

  const void* context = nullptr;  // F_{t-1}, also used by the decoder part below
  NC_HIP(ctx, temporal_context(ctx, &context), "feature extractor");

  void* z = ctx->p(L.zA);
  bool down_done = false;  // the downsample ran inside the encoder's block chain
  PwArgs a;
  if (ctx->is_int()) {
    a = conv_args(ctx, L.pe, 192, C, P8);
    a.src0 = d_frame;
    a.dst = ctx->p(L.ed);
    a.Cdst = C;
    NC_HIP(ctx, pw(ctx, "embed", LD_FRAME, EP_NHWC, a), "patch embed");
    a = conv_args(ctx, L.fuse_enc, 2 * C, C, P8);
    a.src0 = ctx->p(L.ed);
    a.C0 = C;
  } else {
    // patch embed and fuse as one conv on [u; F] (weights composed at load)
    a = conv_args(ctx, L.enc_in, 192 + C, C, P8);
    a.src0 = d_frame;
  }
  a.src1 = context;
  a.C1 = C;
  a.dst = z;
  a.Cdst = C;
  NC_HIP(ctx, pw(ctx, ctx->is_int() ? "fuse" : "embed_fuse", ctx->is_int() ? LD_NHWC : LD_FRAME_CTX, EP_NHWC, a),
         "fuse_enc");

  {
    std::vector<const void*> srcs;
    std::vector<void*> dsts;
    for (int k = 0; k < c.n_enc_blocks; ++k) {
      void* dst = z == ctx->p(L.zA) ? ctx->p(L.zB) : ctx->p(L.zA);
      srcs.push_back(z);
      dsts.push_back(dst);
      z = dst;
    }
    NC_HIP(ctx, run_blocks(ctx, L.enc, srcs, dsts, &L.down, ctx->p(L.y), &down_done), "encoder blocks");
  }

  if (!down_done) {
    a = conv_args(ctx, L.down, 4 * C, C, P16);
    a.src0 = z;
    a.Csrc = C;
    a.dst = ctx->p(L.y);
    a.Cdst = C;
    NC_HIP(ctx, pw(ctx, "down", LD_DOWN, EP_NHWC, a), "downsample");
  }

  double* const parts = ctx->p<double>(L.partials);
  int np_z = 0;
  if (c.hyperprior) {
    NC_HIP(ctx, z_encode(ctx, d_q + (size_t)C * P16, parts, &np_z), "hyper-analysis");
    NC_HIP(ctx, hyper_synth(ctx), "hyper-synthesis");
  }
  PriorArgs pa;
  std::memset(&pa, 0, sizeof(pa));
  pa.wfrag = ctx->p(L.head.w);
  pa.wfrag_lo = ctx->is_int() ? ctx->p(L.head.wlo) : nullptr;
  pa.bias = ctx->p(L.head.bias);
  pa.yhat_prev = ctx->p(L.yhat[cur]);
  pa.y = ctx->p(L.y);
  pa.q_out = d_q;
  pa.yhat_new = ctx->p(L.yhat[nxt]);
  pa.partials = parts + np_z;
  pa.sigma_tab = ctx->is_int() ? ctx->p<float>(L.sigma_tab) : nullptr;
  pa.k_out = d_k;
  pa.scales = ctx->p<float>(L.c_scales);
  pa.k_tab = ctx->is_int() ? ctx->p<uint8_t>(L.c_ktab) : nullptr;
  pa.C = C;
  pa.P = P16;
  pa.decode = 0;
  if (c.hyperprior) step1_fields(ctx, pa);
  NC_HIP(ctx, prior(ctx, pa, nullptr), "prior/quantise");
  // every rate partial of the frame: z's, then the one or two prior launches'
  int n_parts = np_z + prior_parts(P16, 2 * C);
  if (c.hyperprior) {
    PriorArgs p2 = step2_args(ctx, nxt, 0);
    p2.y = ctx->p(L.y);
    p2.q_out = d_q;
    p2.k_out = d_k;
    p2.partials = parts + n_parts;
    n_parts += prior_parts(P16, C);
    NC_HIP(ctx, prior(ctx, p2, nullptr), "second step");
  }
  if constexpr (!std::is_same<Hook, std::nullptr_t>::value) {
    st = after_prior();
    if (st) return st;
  }

  // the decoder part; its upsample adds up the partials into d_bits
  st = run_decoder(ctx, nxt, d_bits, n_parts);
  return st;
}

// The decode after yhat_t is in place: decoder transform, reconstruction
// generation on f_t (into ed, free after the decoder), reconstruction conv.
ncodec_status decode_tail(ncodec_ctx* ctx, void* d_frame_out) {
  const ncodec_config& c = ctx->cfg;
  const int C = c.channels;
  const int P8 = (c.height / 8) * (c.width / 8);
  const Layout& L = ctx->L;
  const int nxt = 1 - ctx->cur;
  ncodec_status st = run_decoder(ctx, nxt);
  if (st) return st;
  const void* rsrc = nullptr;
  NC_HIP(ctx, run_chain(ctx, L.rg, ctx->p(L.feat[nxt]), ctx->p(L.ed), &rsrc), "reconstruction generation");
  PwArgs a = conv_args(ctx, L.rec, C, 192, P8);
  a.src0 = rsrc;
  a.C0 = C;
  a.dst = d_frame_out;
  NC_HIP(ctx, pw(ctx, "recon", LD_NHWC, EP_REC, a), "reconstruction");
  return NCODEC_OK;
}

// Enqueues one decode on ctx->stream (or records it under capture).
ncodec_status enqueue_decode(ncodec_ctx* ctx, const int16_t* d_q, void* d_frame_out) {
  const ncodec_config& c = ctx->cfg;
  const int C = c.channels;
  const int P8 = (c.height / 8) * (c.width / 8), P16 = P8 / 4;
  const Layout& L = ctx->L;
  const int cur = ctx->cur, nxt = 1 - cur;

  PriorArgs pa;
  std::memset(&pa, 0, sizeof(pa));
  pa.wfrag = ctx->p(L.head.w);
  pa.wfrag_lo = ctx->is_int() ? ctx->p(L.head.wlo) : nullptr;
  pa.bias = ctx->p(L.head.bias);
  pa.yhat_prev = ctx->p(L.yhat[cur]);
  pa.q_in = d_q;
  pa.yhat_new = ctx->p(L.yhat[nxt]);
  pa.C = C;
  pa.P = P16;
  pa.decode = 1;
  const void* context = nullptr;
  NC_HIP(ctx, temporal_context(ctx, &context), "feature extractor");
  if (c.hyperprior) {
    NC_HIP(ctx, z_from_symbols(ctx, d_q + (size_t)C * P16), "zhat");
    NC_HIP(ctx, hyper_synth(ctx), "hyper-synthesis");
    step1_fields(ctx, pa);
  }
  NC_HIP(ctx, prior(ctx, pa, nullptr), "prior (decode)");
  if (c.hyperprior) {
    PriorArgs p2 = step2_args(ctx, nxt, 1);
    p2.q_in = d_q;
    NC_HIP(ctx, prior(ctx, p2, nullptr), "second step (decode)");
  }
  return decode_tail(ctx, d_frame_out);
}

const uint16_t* rans_tab(const ncodec_ctx* ctx) { return ctx->p<uint16_t>(ctx->L.c_tab); }

// Scale indices of the next frame's symbols, from the current state (the
// prior head on yhat_{t-1}, Supp. B.2), into d_k (planar, C x h16 x w16).
ncodec_status enqueue_scales(ncodec_ctx* ctx, uint8_t* d_k, void* mu_out = nullptr) {
  const int C = ctx->cfg.channels;
  const int P16 = (ctx->cfg.height / 16) * (ctx->cfg.width / 16);
  const Layout& L = ctx->L;
  PriorArgs pa;
  std::memset(&pa, 0, sizeof(pa));
  pa.wfrag = ctx->p(L.head.w);
  pa.wfrag_lo = ctx->is_int() ? ctx->p(L.head.wlo) : nullptr;
  pa.bias = ctx->p(L.head.bias);
  pa.yhat_prev = ctx->p(L.yhat[ctx->cur]);
  pa.k_out = d_k;
  pa.scales = ctx->p<float>(L.c_scales);
  pa.k_tab = ctx->is_int() ? ctx->p<uint8_t>(L.c_ktab) : nullptr;
  pa.mu_out = mu_out;
  pa.C = C;
  pa.P = P16;
  pa.decode = 2;
  NC_HIP(ctx, prior(ctx, pa, nullptr), "prior (scale indices)");
  return NCODEC_OK;
}

size_t stream_capacity(int64_t n) {
  const int64_t ns = (n + kRansStream - 1) / kRansStream;
  return (size_t)rans_payload_offset((int)ns) + (size_t)ns * kRansMaxWords * 2;
}

// Replaces one pointer in the argument struct of a captured kernel node.
template <class T, class F>
hipError_t set_struct_arg(hipGraphExec_t x, hipGraphNode_t n, F&& edit) {
  hipKernelNodeParams p;
  hipError_t e = hipGraphKernelNodeGetParams(n, &p);
  if (e != hipSuccess) return e;
  if (!p.kernelParams) return hipErrorInvalidValue;
  T v;
  std::memcpy(&v, p.kernelParams[0], sizeof(T));
  edit(v);
  void* args[1] = {&v};
  p.kernelParams = args;
  p.extra = nullptr;
  return hipGraphExecKernelNodeSetParams(x, n, &p);
}

// Replaces the first (pointer) argument of a captured kernel node whose
// arguments are not a struct (the zhat kernel of the two-step model).
hipError_t set_first_ptr_arg(hipGraphExec_t x, hipGraphNode_t n, const void* ptr) {
  hipKernelNodeParams p;
  hipError_t e = hipGraphKernelNodeGetParams(n, &p);
  if (e != hipSuccess) return e;
  if (!p.kernelParams) return hipErrorInvalidValue;
  // the zhat kernel takes 7 arguments: q, mu, yhat, C, P, ld, c_off
  void* args[7];
  for (int i = 0; i < 7; ++i) args[i] = p.kernelParams[i];
  args[0] = &ptr;
  p.kernelParams = args;
  p.extra = nullptr;
  return hipGraphExecKernelNodeSetParams(x, n, &p);
}

// Points the caller-buffer nodes of a captured graph at this call's buffers:
// encode ptr = {frame, q, bits}, decode ptr = {q, frame_out}.  With the
// two-step model the z symbols follow y's in q: the z quantiser (encode) and
// the zhat kernel (decode) take q + C H/16 W/16.
hipError_t retarget(ncodec_ctx* ctx, ncodec_ctx::GraphSlot& gs, bool decode, const void* const* ptr) {
  hipError_t e = hipSuccess;
  for (const auto& cn : gs.nodes) {
    if (e != hipSuccess) break;
    if (!decode && (!std::strcmp(cn.kind, "embed") || !std::strcmp(cn.kind, "embed_fuse")) && ptr[0] != gs.ptr[0]) {
      e = set_struct_arg<PwArgs>(gs.exec, cn.node, [&](PwArgs& v) { v.src0 = ptr[0]; });
    } else if (!std::strcmp(cn.kind, "prior") && ptr[decode ? 0 : 1] != gs.ptr[decode ? 0 : 1]) {
      int16_t* q = (int16_t*)ptr[decode ? 0 : 1];
      e = set_struct_arg<PwArgs>(gs.exec, cn.node, [&](PwArgs& v) {
        if (decode) {
          v.q_in = q;
        } else {
          v.q_out = q;
        }
      });
    } else if (!std::strcmp(cn.kind, decode ? "zhat" : "zquant") && ptr[decode ? 0 : 1] != gs.ptr[decode ? 0 : 1]) {
      int16_t* qz = (int16_t*)ptr[decode ? 0 : 1] + (size_t)ctx->cfg.channels * P16_of(ctx);
      e = decode ? set_first_ptr_arg(gs.exec, cn.node, qz)
                 : set_struct_arg<PwArgs>(gs.exec, cn.node, [&](PwArgs& v) { v.q_out = qz; });
    } else if (!decode && (!std::strcmp(cn.kind, "up") || !std::strcmp(cn.kind, "up_fuse")) && ptr[2] != gs.ptr[2]) {
      e = set_struct_arg<PwArgs>(gs.exec, cn.node, [&](PwArgs& v) { if (v.bits_out) v.bits_out = (double*)ptr[2]; });
    } else if (decode && !std::strcmp(cn.kind, "recon") && ptr[1] != gs.ptr[1]) {
      e = set_struct_arg<PwArgs>(gs.exec, cn.node, [&](PwArgs& v) { v.dst = (void*)ptr[1]; });
    }
  }
  if (e == hipSuccess) for (int i = 0; i < 3; ++i) gs.ptr[i] = ptr[i];
  return e;
}

// Runs one encode or decode as a graph replay: the first call for a state
// parity captures the launch sequence (on a private stream, so the caller's
// stream may be the null stream), later calls only retarget caller buffers.
ncodec_status run_graph(ncodec_ctx* ctx, bool decode, const void* p0, const void* p1, const void* p2) {
  ncodec_ctx::GraphSlot& gs = ctx->graphs[decode][ctx->cur];
  const void* ptr[3] = {p0, p1, p2};
  if (!gs.exec) {
    if (!ctx->cap_stream) NC_HIP(ctx, hipStreamCreateWithFlags(&ctx->cap_stream, hipStreamNonBlocking), "capture stream");
    const hipStream_t user = ctx->stream;
    ctx->stream = ctx->cap_stream;
    gs.nodes.clear();
    ctx->capturing = &gs.nodes;
    hipError_t e = hipStreamBeginCapture(ctx->cap_stream, hipStreamCaptureModeThreadLocal);
    ncodec_status st = NCODEC_OK;
    if (e == hipSuccess) {
      st = decode ? enqueue_decode(ctx, (const int16_t*)p0, (void*)p1)
                  : enqueue_encode(ctx, p0, (int16_t*)p1, (double*)p2);
      hipGraph_t g = nullptr;
      const hipError_t e2 = hipStreamEndCapture(ctx->cap_stream, &g);
      gs.graph = g;
      if (e2 != hipSuccess && st == NCODEC_OK) st = hip_fail(ctx, e2, "graph capture");
    } else {
      st = hip_fail(ctx, e, "begin graph capture");
    }
    ctx->capturing = nullptr;
    ctx->stream = user;
    if (st == NCODEC_OK) {
      e = hipGraphInstantiate(&gs.exec, gs.graph, nullptr, nullptr, 0);
      if (e != hipSuccess) st = hip_fail(ctx, e, "graph instantiate");
    }
    if (st != NCODEC_OK) {
      if (gs.graph) (void)hipGraphDestroy(gs.graph);
      gs = ncodec_ctx::GraphSlot{};
      return st;
    }
    for (int i = 0; i < 3; ++i) gs.ptr[i] = ptr[i];
  } else {
    NC_HIP(ctx, retarget(ctx, gs, decode, ptr), "graph update");
  }
  NC_HIP(ctx, hipGraphLaunch(gs.exec, ctx->stream), "graph launch");
  return NCODEC_OK;
}

// The second stream and its two events, created on first use.
ncodec_status ensure_aux(ncodec_ctx* ctx) {
  if (!ctx->aux) NC_HIP(ctx, hipStreamCreateWithFlags(&ctx->aux, hipStreamNonBlocking), "aux stream");
  if (!ctx->ev_fork) NC_HIP(ctx, hipEventCreateWithFlags(&ctx->ev_fork, hipEventDisableTiming), "fork event");
  if (!ctx->ev_join) NC_HIP(ctx, hipEventCreateWithFlags(&ctx->ev_join, hipEventDisableTiming), "join event");
  return NCODEC_OK;
}

}  // namespace

extern "C" {

size_t ncodec_weight_count(const ncodec_config* cfg) {
  if (!cfg_valid(cfg, nullptr)) return 0;
  return weight_count(*cfg);
}

size_t ncodec_workspace_bytes(const ncodec_config* cfg) {
  if (!cfg_valid(cfg, nullptr)) return 0;
  Image img;
  Layout L;
  build_layout(*cfg, nullptr, img, L, nullptr);
  return L.total;
}

ncodec_status ncodec_create(const ncodec_config* cfg, const float* host_weights, size_t n_weights, void* d_workspace,
                            size_t ws_bytes, void* hip_stream, ncodec_ctx** out) {
  std::string why;
  if (!out) return fail(nullptr, NCODEC_EINVAL, "out is NULL");
  *out = nullptr;
  if (!cfg) return fail(nullptr, NCODEC_EINVAL, "cfg is NULL");
  if (!cfg_valid(cfg, &why)) return fail(nullptr, NCODEC_ESHAPE, why);
  if (!host_weights) return fail(nullptr, NCODEC_EINVAL, "host_weights is NULL");
  if (n_weights != weight_count(*cfg))
    return fail(nullptr, NCODEC_EINVAL,
                "n_weights is " + std::to_string(n_weights) + ", expected " + std::to_string(weight_count(*cfg)));
  if (!d_workspace) return fail(nullptr, NCODEC_EINVAL, "d_workspace is NULL");
  if ((uintptr_t)d_workspace % kAlign) return fail(nullptr, NCODEC_ENOMEM, "d_workspace must be 256-byte aligned");
  for (size_t i = 0; i < n_weights; ++i)
    if (!std::isfinite(host_weights[i])) return fail(nullptr, NCODEC_EINVAL, "non-finite weight");

  Image img;
  Layout L;
  if (!build_layout(*cfg, host_weights, img, L, &why)) return fail(nullptr, NCODEC_EINVAL, why);
  if (ws_bytes < L.total)
    return fail(nullptr, NCODEC_ENOMEM,
                "workspace has " + std::to_string(ws_bytes) + " bytes, needs " + std::to_string(L.total));

  ncodec_ctx* ctx = new ncodec_ctx();
  ctx->cfg = *cfg;
  if (cfg->qp_banks || cfg->hyperprior) ctx->host_w.assign(host_weights, host_weights + n_weights);
  ctx->stream = (hipStream_t)hip_stream;
  ctx->ws = (char*)d_workspace;
  ctx->L = std::move(L);
  hipError_t e = hipGetDevice(&ctx->device);
  if (e == hipSuccess) e = hipMemcpyAsync(ctx->ws, img.bytes.data(), img.bytes.size(), hipMemcpyHostToDevice, ctx->stream);
  if (e == hipSuccess) e = launch_fill_zero(ctx->ws + ctx->L.image_bytes, ctx->L.total - ctx->L.image_bytes, ctx->stream);
  if (e == hipSuccess) e = hipStreamSynchronize(ctx->stream);
  if (e != hipSuccess) {
    g_create_error = std::string("create: ") + hipGetErrorString(e);
    delete ctx;
    return NCODEC_EHIP;
  }
  *out = ctx;
  return NCODEC_OK;
}

ncodec_status ncodec_set_qp(ncodec_ctx* ctx, int32_t qp) {
  if (ctx && (qp < 0 || qp >= kNumQp)) return fail(ctx, NCODEC_EINVAL, "qp must be in [0, 64)");
  return ncodec_set_rate(ctx, (double)qp);
}

ncodec_status ncodec_set_rate(ncodec_ctx* ctx, double qp) {
  ncodec_status st = enter(ctx);
  if (st) return st;
  if (!ctx->cfg.qp_banks && !ctx->cfg.hyperprior)
    return fail(ctx, NCODEC_EINVAL, "the context has no rate banks (qp_banks = 0, hyperprior = 0)");
  if (!(qp >= 0.0 && qp <= kNumQp - 1)) return fail(ctx, NCODEC_EINVAL, "qp must be in [0, 63]");
  if (qp == ctx->qp) return NCODEC_OK;
  Image img;
  Layout L;
  std::string why;
  if (!build_layout(ctx->cfg, ctx->host_w.data(), img, L, &why, qp)) return fail(ctx, NCODEC_EINVAL, why);
  if (L.image_bytes != ctx->L.image_bytes) return fail(ctx, NCODEC_EINVAL, "internal: image size depends on qp");
  NC_HIP(ctx, hipMemcpyAsync(ctx->ws, img.bytes.data(), img.bytes.size(), hipMemcpyHostToDevice, ctx->stream),
         "set_rate upload");
  NC_HIP(ctx, hipStreamSynchronize(ctx->stream), "set_rate");
  ctx->qp = qp;
  return NCODEC_OK;
}

ncodec_status ncodec_reset(ncodec_ctx* ctx) {
  ncodec_status st = enter(ctx);
  if (st) return st;
  const int C = ctx->cfg.channels;
  const size_t P8 = (size_t)(ctx->cfg.height / 8) * (ctx->cfg.width / 8);
  NC_HIP(ctx, launch_fill_zero(ctx->p(ctx->L.feat[ctx->cur]), P8 * C * 2, ctx->stream), "reset");
  NC_HIP(ctx, launch_fill_zero(ctx->p(ctx->L.yhat[ctx->cur]), P8 / 4 * C * 2, ctx->stream), "reset");
  return NCODEC_OK;
}

ncodec_status ncodec_encode_frame(ncodec_ctx* ctx, const void* d_frame, int16_t* d_q, double* d_bits) {
  ncodec_status st = enter(ctx);
  if (st) return st;
  if (!d_frame || !d_q) return fail(ctx, NCODEC_EINVAL, "d_frame and d_q must be non-NULL");
  if ((uintptr_t)d_frame % 16 || (uintptr_t)d_q % 16) return fail(ctx, NCODEC_EINVAL, "d_frame and d_q must be 16-byte aligned");
  ncodec_status st2;
  if (ctx->use_graphs && !ctx->timing)
    st2 = run_graph(ctx, false, d_frame, d_q, d_bits ? (const void*)d_bits : ctx->p(ctx->L.spare_bits));
  else
    st2 = enqueue_encode(ctx, d_frame, d_q, d_bits);
  if (st2) return st2;
  ctx->cur = 1 - ctx->cur;
  return NCODEC_OK;
}

ncodec_status ncodec_decode_frame(ncodec_ctx* ctx, const int16_t* d_q, void* d_frame_out) {
  ncodec_status st = enter(ctx);
  if (st) return st;
  if (!d_q || !d_frame_out) return fail(ctx, NCODEC_EINVAL, "d_q and d_frame_out must be non-NULL");
  if ((uintptr_t)d_frame_out % 16 || (uintptr_t)d_q % 16)
    return fail(ctx, NCODEC_EINVAL, "d_q and d_frame_out must be 16-byte aligned");
  ncodec_status st2;
  if (ctx->use_graphs && !ctx->timing)
    st2 = run_graph(ctx, true, d_q, d_frame_out, nullptr);
  else
    st2 = enqueue_decode(ctx, d_q, d_frame_out);
  if (st2) return st2;
  ctx->cur = 1 - ctx->cur;
  return NCODEC_OK;
}

ncodec_status ncodec_estimate_bits(ncodec_ctx* ctx, const int16_t* d_q, const void* d_scale, int64_t n,
                                   double* d_bits) {
  ncodec_status st = enter(ctx);
  if (st) return st;
  if (!d_bits) return fail(ctx, NCODEC_EINVAL, "d_bits is NULL");
  if (n < 0 || n >= ((int64_t)1 << 31)) return fail(ctx, NCODEC_EINVAL, "n out of range");
  if (n > 0 && (!d_q || !d_scale)) return fail(ctx, NCODEC_EINVAL, "d_q and d_scale must be non-NULL");
  const float* tab = ctx->is_int() ? ctx->p<float>(ctx->L.sigma_tab) : nullptr;
  NC_HIP(ctx, launch_estimate_bits(d_q, d_scale, tab, n, ctx->p<double>(ctx->L.partials), d_bits, ctx->stream),
         "estimate_bits");
  return NCODEC_OK;
}

size_t ncodec_stream_capacity(const ncodec_config* cfg) {
  if (!cfg_valid(cfg, nullptr)) return 0;
  const int64_t ny = (int64_t)(cfg->height / 16) * (cfg->width / 16) * cfg->channels;
  if (!cfg->hyperprior) return stream_capacity(ny);
  const int64_t nz = (int64_t)(cfg->height / 32) * (cfg->width / 32) * kCZ;
  return stream_capacity(nz) + 2 * stream_capacity(ny / 2);
}

size_t ncodec_symbol_count(const ncodec_config* cfg) {
  if (!cfg_valid(cfg, nullptr)) return 0;
  const size_t ny = (size_t)(cfg->height / 16) * (cfg->width / 16) * cfg->channels;
  return ny + (cfg->hyperprior ? (size_t)(cfg->height / 32) * (cfg->width / 32) * kCZ : 0);
}

ncodec_status ncodec_scale_indices(ncodec_ctx* ctx, uint8_t* d_k) {
  ncodec_status st = enter(ctx);
  if (st) return st;
  if (!d_k) return fail(ctx, NCODEC_EINVAL, "d_k is NULL");
  if (ctx->cfg.hyperprior)
    return fail(ctx, NCODEC_ESTATE, "scale indices depend on the frame's z and y^1 with the two-step entropy model");
  return enqueue_scales(ctx, d_k);
}

ncodec_status ncodec_rans_encode(ncodec_ctx* ctx, const int16_t* d_q, const uint8_t* d_k, int64_t n, void* d_stream,
                                 size_t capacity, uint64_t* d_stream_bytes) {
  ncodec_status st = enter(ctx);
  if (st) return st;
  if (n <= 0 || n > ctx->L.n_sym) return fail(ctx, NCODEC_EINVAL, "n must be in [1, symbols per frame]");
  if (!d_q || !d_k || !d_stream || !d_stream_bytes) return fail(ctx, NCODEC_EINVAL, "NULL buffer");
  if ((uintptr_t)d_stream % 4) return fail(ctx, NCODEC_EINVAL, "d_stream must be 4-byte aligned");
  if ((uintptr_t)d_q % 16 || (uintptr_t)d_k % 16) return fail(ctx, NCODEC_EINVAL, "d_q and d_k must be 16-byte aligned");
  if (capacity < stream_capacity(n))
    return fail(ctx, NCODEC_EINVAL, "capacity below the worst case of " + std::to_string(stream_capacity(n)) + " bytes");
  const Layout& L = ctx->L;
  NC_HIP(ctx, timed(ctx, "rans_enc", [&] {
           return launch_rans_encode(d_q, d_k, n, rans_tab(ctx), ctx->p<uint16_t>(L.rscratch), kRansMaxWords,
                                     ctx->p<uint32_t>(L.rlens), (uint8_t*)d_stream, d_stream_bytes, ctx->stream);
         }),
         "rans encode");
  return NCODEC_OK;
}

ncodec_status ncodec_rans_decode(ncodec_ctx* ctx, const void* d_stream, size_t stream_bytes, const uint8_t* d_k,
                                 int64_t n, int16_t* d_q, int32_t* d_status) {
  ncodec_status st = enter(ctx);
  if (st) return st;
  if (n <= 0 || n > ctx->L.n_sym) return fail(ctx, NCODEC_EINVAL, "n must be in [1, symbols per frame]");
  if (!d_stream || !d_k || !d_q) return fail(ctx, NCODEC_EINVAL, "NULL buffer");
  if ((uintptr_t)d_stream % 4) return fail(ctx, NCODEC_EINVAL, "d_stream must be 4-byte aligned");
  if ((uintptr_t)d_k % 16) return fail(ctx, NCODEC_EINVAL, "d_k must be 16-byte aligned");
  const Layout& L = ctx->L;
  NC_HIP(ctx, timed(ctx, "rans_dec", [&] {
           return launch_rans_decode((const uint8_t*)d_stream, stream_bytes, d_k, n, rans_tab(ctx),
                                     ctx->p<uint32_t>(L.rerrs), ctx->p<uint32_t>(L.rcount), d_q, d_status, ctx->stream);
         }),
         "rans decode");
  return NCODEC_OK;
}

ncodec_status ncodec_encode_frame_coded(ncodec_ctx* ctx, const void* d_frame, int16_t* d_q, double* d_bits,
                                        void* d_stream, size_t capacity, uint64_t* d_stream_bytes) {
  ncodec_status st = enter(ctx);
  if (st) return st;
  if (!d_frame || !d_stream || !d_stream_bytes) return fail(ctx, NCODEC_EINVAL, "NULL buffer");
  if ((uintptr_t)d_frame % 16 || (d_q && (uintptr_t)d_q % 16)) return fail(ctx, NCODEC_EINVAL, "d_frame and d_q must be 16-byte aligned");
  if ((uintptr_t)d_stream % 4) return fail(ctx, NCODEC_EINVAL, "d_stream must be 4-byte aligned");
  const Layout& L = ctx->L;
  if (capacity < ncodec_stream_capacity(&ctx->cfg))
    return fail(ctx, NCODEC_EINVAL, "capacity below ncodec_stream_capacity()");
  const bool par = ctx->overlap;
  if (par && (st = ensure_aux(ctx))) return st;
  int16_t* q = d_q ? d_q : ctx->p<int16_t>(L.qtmp);
  // one container: all symbols; two-step model: z, y^1, y^2 at fixed offsets
  auto section = [&](hipStream_t s, const int16_t* sq, const uint8_t* sk, int64_t n, size_t off,
                     uint64_t* nbytes) -> ncodec_status {
    NC_HIP(ctx, timed(ctx, "rans_enc", [&] {
             return launch_rans_encode(sq, sk, n, rans_tab(ctx), ctx->p<uint16_t>(L.rscratch), kRansMaxWords,
                                       ctx->p<uint32_t>(L.rlens), (uint8_t*)d_stream + off, nbytes, s);
           }),
           "rans encode");
    return NCODEC_OK;
  };
  // the coder: on the context's stream after the decoder, or (parallel coding)
  // on the second stream as soon as q and the scale indices exist, while the
  // decoder part of the encode runs (Fig. 6)
  auto coder = [&](hipStream_t s) -> ncodec_status {
    const uint8_t* k = ctx->p<uint8_t>(L.kmap);
    if (!ctx->cfg.hyperprior) return section(s, q, k, L.n_sym, 0, d_stream_bytes);
    const int64_t nh = L.n_sym / 2;
    const size_t c0 = stream_capacity(L.n_z), c1 = stream_capacity(nh);
    ncodec_status s2 = section(s, q + L.n_sym, ctx->p<uint8_t>(L.zk), L.n_z, 0, d_stream_bytes);
    if (!s2) s2 = section(s, q, k, nh, c0, d_stream_bytes + 1);
    if (!s2) s2 = section(s, q + nh, k + nh, nh, c0 + c1, d_stream_bytes + 2);
    return s2;
  };
  if (par) {
    st = enqueue_encode(ctx, d_frame, q, d_bits, ctx->p<uint8_t>(L.kmap), [&]() -> ncodec_status {
      NC_HIP(ctx, hipEventRecord(ctx->ev_fork, ctx->stream), "fork");
      NC_HIP(ctx, hipStreamWaitEvent(ctx->aux, ctx->ev_fork, 0), "fork");
      ncodec_status s2 = coder(ctx->aux);
      if (s2) return s2;
      NC_HIP(ctx, hipEventRecord(ctx->ev_join, ctx->aux), "join");
      return NCODEC_OK;
    });
    if (st) return st;
    NC_HIP(ctx, hipStreamWaitEvent(ctx->stream, ctx->ev_join, 0), "join");
  } else {
    st = enqueue_encode(ctx, d_frame, q, d_bits, ctx->p<uint8_t>(L.kmap));
    if (st) return st;
    st = coder(ctx->stream);
    if (st) return st;
  }
  ctx->cur = 1 - ctx->cur;
  return NCODEC_OK;
}

ncodec_status ncodec_decode_frame_coded(ncodec_ctx* ctx, const void* d_stream, size_t stream_bytes, void* d_frame_out,
                                        int32_t* d_status) {
  ncodec_status st = enter(ctx);
  if (st) return st;
  if (!d_stream || !d_frame_out) return fail(ctx, NCODEC_EINVAL, "NULL buffer");
  if ((uintptr_t)d_frame_out % 16) return fail(ctx, NCODEC_EINVAL, "d_frame_out must be 16-byte aligned");
  if ((uintptr_t)d_stream % 4) return fail(ctx, NCODEC_EINVAL, "d_stream must be 4-byte aligned");
  const Layout& L = ctx->L;
  const int C = ctx->cfg.channels;
  const int P16 = (ctx->cfg.height / 16) * (ctx->cfg.width / 16);
  // the feature extractor does not depend on the symbols: with parallel coding
  // it runs on the second stream while the symbols are decoded (Fig. 6)
  const bool par = ctx->overlap && !L.fe.empty();
  if (par && (st = ensure_aux(ctx))) return st;
  const void* context = nullptr;
  if (par) {
    NC_HIP(ctx, hipEventRecord(ctx->ev_fork, ctx->stream), "fork");
    NC_HIP(ctx, hipStreamWaitEvent(ctx->aux, ctx->ev_fork, 0), "fork");
    const hipStream_t user = ctx->stream;
    ctx->stream = ctx->aux;
    const hipError_t e = temporal_context(ctx, &context);
    ctx->stream = user;
    NC_HIP(ctx, e, "feature extractor");
    NC_HIP(ctx, hipEventRecord(ctx->ev_join, ctx->aux), "join");
  } else {
    NC_HIP(ctx, temporal_context(ctx, &context), "feature extractor");
  }
  auto ad = [&](size_t off, size_t bytes, const uint8_t* k, int64_t n, int16_t* q, int32_t* status) -> hipError_t {
    return timed(ctx, "rans_dec", [&] {
      return launch_rans_decode((const uint8_t*)d_stream + off, bytes, k, n, rans_tab(ctx), ctx->p<uint32_t>(L.rerrs),
                                ctx->p<uint32_t>(L.rcount), q, status, ctx->stream);
    });
  };
  auto yhat = [&](const int16_t* q, int nch, int c_off) -> hipError_t {
    return timed(ctx, "yhat", [&] {
      return launch_yhat_from_q(q, ctx->p(L.mu), ctx->p(L.yhat[1 - ctx->cur]), nch, P16, ctx->is_int(), ctx->stream,
                                C, c_off);
    });
  };
  int16_t* const qt = ctx->p<int16_t>(L.qtmp);
  uint8_t* const kt = ctx->p<uint8_t>(L.kmap);
  if (!ctx->cfg.hyperprior) {
    // one prior pass: the scale indices for the coder and mu for yhat = q + mu
    st = enqueue_scales(ctx, kt, ctx->p(L.mu));
    if (st) return st;
    NC_HIP(ctx, ad(0, stream_bytes, kt, L.n_sym, qt, d_status), "rans decode");
    NC_HIP(ctx, yhat(qt, C, 0), "yhat");
  } else {
    // z, then its hyper parameters and the first step's distribution, y^1,
    // then the second step's distribution, y^2 (supplementary "Parallel Coding")
    const int64_t nh = L.n_sym / 2;
    const size_t c0 = stream_capacity(L.n_z), c1 = stream_capacity(nh);
    if (stream_bytes < c0 + 2 * c1) return fail(ctx, NCODEC_EINVAL, "stream_bytes below ncodec_stream_capacity()");
    const int nxt = 1 - ctx->cur;
    NC_HIP(ctx, ad(0, c0, ctx->p<uint8_t>(L.zk), L.n_z, qt + L.n_sym, d_status), "rans decode (z)");
    NC_HIP(ctx, z_from_symbols(ctx, qt + L.n_sym), "zhat");
    NC_HIP(ctx, hyper_synth(ctx), "hyper-synthesis");
    PriorArgs pa;
    std::memset(&pa, 0, sizeof(pa));
    pa.wfrag = ctx->p(L.head.w);
    pa.wfrag_lo = ctx->is_int() ? ctx->p(L.head.wlo) : nullptr;
    pa.bias = ctx->p(L.head.bias);
    pa.yhat_prev = ctx->p(L.yhat[ctx->cur]);
    pa.k_out = kt;
    pa.mu_out = ctx->p(L.mu);
    pa.scales = ctx->p<float>(L.c_scales);
    pa.k_tab = ctx->is_int() ? ctx->p<uint8_t>(L.c_ktab) : nullptr;
    pa.C = C;
    pa.P = P16;
    pa.decode = 2;
    step1_fields(ctx, pa);
    NC_HIP(ctx, prior(ctx, pa, nullptr), "prior (scale indices, step 1)");
    NC_HIP(ctx, ad(c0, c1, kt, nh, qt, d_status ? d_status + 1 : nullptr), "rans decode (y^1)");
    NC_HIP(ctx, yhat(qt, C / 2, 0), "yhat^1");
    PriorArgs p2 = step2_args(ctx, nxt, 2);
    p2.k_out = kt;
    p2.mu_out = ctx->p(L.mu);
    NC_HIP(ctx, prior(ctx, p2, nullptr), "prior (scale indices, step 2)");
    NC_HIP(ctx, ad(c0 + c1, c1, kt + nh, nh, qt + nh, d_status ? d_status + 2 : nullptr), "rans decode (y^2)");
    NC_HIP(ctx, yhat(qt + nh, C / 2, C / 2), "yhat^2");
  }
  if (par) NC_HIP(ctx, hipStreamWaitEvent(ctx->stream, ctx->ev_join, 0), "join");
  st = decode_tail(ctx, d_frame_out);
  if (st) return st;
  ctx->cur = 1 - ctx->cur;
  return NCODEC_OK;
}

ncodec_status ncodec_parallel_coding(ncodec_ctx* ctx, int32_t enable) {
  ncodec_status st = enter(ctx);
  if (st) return st;
  ctx->overlap = enable != 0;
  return NCODEC_OK;
}

ncodec_status ncodec_get_state(ncodec_ctx* ctx, void* d_feat, void* d_yhat) {
  ncodec_status st = enter(ctx);
  if (st) return st;
  const int C = ctx->cfg.channels;
  const int P8 = (ctx->cfg.height / 8) * (ctx->cfg.width / 8);
  if (d_feat) NC_HIP(ctx, launch_nhwc_to_planar(ctx->p(ctx->L.feat[ctx->cur]), d_feat, C, P8, ctx->stream), "get_state");
  if (d_yhat) NC_HIP(ctx, launch_nhwc_to_planar(ctx->p(ctx->L.yhat[ctx->cur]), d_yhat, C, P8 / 4, ctx->stream), "get_state");
  return NCODEC_OK;
}

ncodec_status ncodec_set_state(ncodec_ctx* ctx, const void* d_feat, const void* d_yhat) {
  ncodec_status st = enter(ctx);
  if (st) return st;
  const int C = ctx->cfg.channels;
  const int P8 = (ctx->cfg.height / 8) * (ctx->cfg.width / 8);
  if (d_feat) NC_HIP(ctx, launch_planar_to_nhwc(d_feat, ctx->p(ctx->L.feat[ctx->cur]), C, P8, ctx->stream), "set_state");
  if (d_yhat) NC_HIP(ctx, launch_planar_to_nhwc(d_yhat, ctx->p(ctx->L.yhat[ctx->cur]), C, P8 / 4, ctx->stream), "set_state");
  return NCODEC_OK;
}

// Launches of a run of n DC blocks (chains: up to kMaxChain blocks each).
int block_launches(ncodec_ctx* ctx, int n) {
  if (n < 2 || !chains_usable(ctx)) return n;
  return (n + kMaxChain - 1) / kMaxChain;
}

// Whether the encoder's last block launch carries the downsample (fp16: its
// last run of blocks is a chain of at least two).
bool down_fused(ncodec_ctx* ctx, int n) {
  return !ctx->is_int() && n >= 2 && chains_usable(ctx) && n - kMaxChain * ((n - 1) / kMaxChain) >= 2;
}

int32_t ncodec_kernels_per_frame(const ncodec_ctx* cctx, int32_t decode) {
  if (!cctx) return 0;
  ncodec_ctx* ctx = const_cast<ncodec_ctx*>(cctx);  // caches the residency check
  const ncodec_config& c = ctx->cfg;
  // feature extractor, prior, upsample, fuse, decoder blocks, reconstruction generation, reconstruction
  // (two-step model: z quantiser or z from symbols, hyper-synthesis, second step)
  // (the fp16 path runs the upsample and the fuse as one launch, and in an
  // encode the patch embed and the fuse too, and the downsample inside the
  // encoder's block chain)
  const int fold = c.path == NCODEC_PATH_INT16 ? 0 : 1;
  const int hyper = c.hyperprior ? 3 : 0;
  const int per_block = c.channels > 256 ? 3 : 1;  // a wide block is three launches
  if (per_block == 1) {  // one launch per block or per chain of blocks
    const int fe = block_launches(ctx, c.n_fe_blocks), dec = block_launches(ctx, c.n_dec_blocks);
    if (decode) return 4 - fold + hyper + fe + dec + block_launches(ctx, c.n_rg_blocks);
    return 6 - 2 * fold + hyper + fe + block_launches(ctx, c.n_enc_blocks) + dec - (down_fused(ctx, c.n_enc_blocks) ? 1 : 0);
  }
  if (decode) return 4 - fold + hyper + per_block * (c.n_fe_blocks + c.n_dec_blocks + c.n_rg_blocks);
  // feature extractor, embed, fuse, encoder blocks, downsample, prior, upsample (with the bit total), fuse,
  // decoder blocks
  return 6 - 2 * fold + hyper + per_block * (c.n_fe_blocks + c.n_enc_blocks + c.n_dec_blocks);
}

ncodec_status ncodec_graph_enable(ncodec_ctx* ctx, int32_t enable) {
  ncodec_status st = enter(ctx);
  if (st) return st;
  ctx->use_graphs = enable != 0;
  return NCODEC_OK;
}

ncodec_status ncodec_block_chains(ncodec_ctx* ctx, int32_t enable) {
  ncodec_status st = enter(ctx);
  if (st) return st;
  if (ctx->chains != (enable != 0)) {
    // captured graphs hold the other launch sequence: capture again on next use
    NC_HIP(ctx, hipStreamSynchronize(ctx->stream), "block_chains");
    for (auto& row : ctx->graphs)
      for (auto& gs : row) {
        if (gs.exec) (void)hipGraphExecDestroy(gs.exec);
        if (gs.graph) (void)hipGraphDestroy(gs.graph);
        gs = ncodec_ctx::GraphSlot{};
      }
  }
  ctx->chains = enable != 0;
  return NCODEC_OK;
}

ncodec_status ncodec_block_chain_status(ncodec_ctx* ctx, int32_t* in_use, int32_t* timeouts) {
  ncodec_status st = enter(ctx);
  if (st) return st;
  if (!in_use || !timeouts) return fail(ctx, NCODEC_EINVAL, "in_use and timeouts must not be NULL");
  *in_use = block_launches(ctx, 2) == 1 ? 1 : 0;
  *timeouts = 0;
  if (!ctx->L.chain_status) return NCODEC_OK;
  int32_t v = 0;
  NC_HIP(ctx, hipMemcpyAsync(&v, ctx->p(ctx->L.chain_status), 4, hipMemcpyDeviceToHost, ctx->stream), "chain status");
  NC_HIP(ctx, hipStreamSynchronize(ctx->stream), "chain status");
  *timeouts = v;
  return NCODEC_OK;
}

ncodec_status ncodec_timing_enable(ncodec_ctx* ctx, int32_t enable) {
  ncodec_status st = enter(ctx);
  if (st) return st;
  ctx->timing = enable != 0;
  return NCODEC_OK;
}

ncodec_status ncodec_timing_read(ncodec_ctx* ctx, ncodec_kernel_timing* out, int32_t max_kinds, int32_t* n_kinds) {
  ncodec_status st = enter(ctx);
  if (st) return st;
  if (!n_kinds || (max_kinds > 0 && !out)) return fail(ctx, NCODEC_EINVAL, "out / n_kinds is NULL");
  NC_HIP(ctx, hipStreamSynchronize(ctx->stream), "timing_read");
  std::vector<ncodec_kernel_timing> agg;
  hipError_t err = hipSuccess;
  for (auto& t : ctx->log) {
    float ms = 0.f;
    if (err == hipSuccess && t.start && t.stop) err = hipEventElapsedTime(&ms, t.start, t.stop);
    size_t i = 0;
    while (i < agg.size() && std::strcmp(agg[i].kind, t.kind) != 0) ++i;
    if (i == agg.size()) {
      ncodec_kernel_timing k;
      std::memset(&k, 0, sizeof(k));
      std::strncpy(k.kind, t.kind, sizeof(k.kind) - 1);
      agg.push_back(k);
    }
    agg[i].launches += t.n;
    agg[i].total_ms += ms;
    if (t.start) (void)hipEventDestroy(t.start);
    if (t.stop) (void)hipEventDestroy(t.stop);
  }
  ctx->log.clear();
  if (err != hipSuccess) return hip_fail(ctx, err, "hipEventElapsedTime");
  *n_kinds = (int32_t)agg.size();
  for (int32_t i = 0; i < max_kinds && i < (int32_t)agg.size(); ++i) out[i] = agg[i];
  return NCODEC_OK;
}

const char* ncodec_last_error(const ncodec_ctx* ctx) {
  return ctx ? ctx->err.c_str() : g_create_error.c_str();
}

const char* ncodec_status_string(ncodec_status st) {
  switch (st) {
    case NCODEC_OK: return "ok";
    case NCODEC_EINVAL: return "invalid argument";
    case NCODEC_ESHAPE: return "invalid shape or configuration";
    case NCODEC_EHIP: return "HIP runtime error";
    case NCODEC_ESTATE: return "call does not match the context";
    case NCODEC_EOVERFLOW: return "int32 accumulator overflow";
    case NCODEC_ENOMEM: return "workspace too small or misaligned";
  }
  return "unknown status";
}

void ncodec_destroy(ncodec_ctx* ctx) {
  if (!ctx) return;
  (void)hipSetDevice(ctx->device);
  (void)hipStreamSynchronize(ctx->stream);
  for (auto& t : ctx->log) {
    if (t.start) (void)hipEventDestroy(t.start);
    if (t.stop) (void)hipEventDestroy(t.stop);
  }
  for (auto& row : ctx->graphs)
    for (auto& gs : row) {
      if (gs.exec) (void)hipGraphExecDestroy(gs.exec);
      if (gs.graph) (void)hipGraphDestroy(gs.graph);
    }
  if (ctx->cap_stream) (void)hipStreamDestroy(ctx->cap_stream);
  if (ctx->aux) {
    (void)hipStreamSynchronize(ctx->aux);
    (void)hipStreamDestroy(ctx->aux);
  }
  if (ctx->ev_fork) (void)hipEventDestroy(ctx->ev_fork);
  if (ctx->ev_join) (void)hipEventDestroy(ctx->ev_join);
  delete ctx;
}

}  // extern "C"
