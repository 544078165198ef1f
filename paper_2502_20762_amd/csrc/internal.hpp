// Host-visible launch interface between the scheduler (api.hip) and the
// kernel translation units.  Not part of the public ABI.
#pragma once
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <string>

#include "../../include/ncodec.h"

namespace nc {

// Records msg as the error that ncodec_last_error(NULL) reports (this thread)
// and returns st.
ncodec_status set_error(ncodec_status st, const std::string& msg);

// Events attached to the next kernel dispatch (timing mode of the C ABI): when
// set, launches go through hipExtLaunchKernelGGL, whose start / stop events
// bracket exactly that dispatch.
struct LaunchEvents {
  hipEvent_t start = nullptr, stop = nullptr;
};
extern thread_local LaunchEvents g_launch_events;

template <typename F, typename... Args>
inline void launch(F kernel, dim3 grid, dim3 block, hipStream_t st, Args... args) {
  if (g_launch_events.start || g_launch_events.stop)
    hipExtLaunchKernelGGL(kernel, grid, block, 0, st, g_launch_events.start, g_launch_events.stop, 0, args...);
  else
    hipLaunchKernelGGL(kernel, grid, block, 0, st, args...);
}

// How a pointwise kernel gathers its activation operand (K index -> memory).
enum Loader : int {
  LD_NHWC = 0,   // k < C0: src0[p*C0 + k], else src1[p*C1 + k - C0]   (concat on channels)
  LD_FRAME = 1,  // planar 3xHxW frame, pixel-unshuffle x8 on load: k = 64c + 8i + j
  LD_DOWN = 2,   // 2x2 stride-2 gather: k = (2i+j)*Csrc + c from pixel (2Y+i, 2X+j)
  // k < 192: the frame as LD_FRAME, else src1[p*C1 + k - 192] (patch embed
  // folded into the encoder's fuse)
  LD_FRAME_CTX = 3,
  // 1/16-scale pixel P, pass of sub-position s = n0 / Cdst: k < C0:
  // src0[P*C0 + k], else src1[child*C1 + k - C0] with child = (2Y + s/2,
  // 2X + s%2) on the 1/8 grid (upsample folded into the decoder's fuse)
  LD_UP_CTX = 4,
};
// Where a pointwise kernel writes its result.
enum Epi : int {
  EP_NHWC = 0,  // dst[p*Cdst + n]
  EP_UP = 1,    // rows ordered (sub-position, channel): pixel-shuffle x2 into the 1/8 grid
  EP_REC = 2,   // rows 64c+8i+j: pixel-shuffle x8 into a planar 3xHxW frame, clamped
  EP_PRIOR = 3,      // rows (32 mu, 32 s) per pass: quantise y, write q, yhat, bit partials
  EP_PRIOR_DEC = 4,  // same rows: yhat = q + mu from the given q
  EP_SCALES = 5,     // same rows: only the scale index of every symbol (entropy decoding)
  EP_ZQUANT = 6,     // 64 rows = the channels of z: q_z = round(z), zhat, rate partials
  EP_LRELU = 7,      // NHWC store of LeakyReLU_0.1(acc + b) (a DC block's hidden layer)
  EP_RESID = 8,      // NHWC store of res + acc + b (a DC block's projection and residual)
  EP_GATE = 9,       // rows (32 h1, 32 h2) per 64: NHWC store of WSiLU(h1) * h2 (gated hidden layer)
};

struct PwArgs {
  const void* wfrag;     // fp16: half8 [N/32][K/16][64]; int: int8x16 hi plane [N/32][K/32][64]
  const void* wfrag_lo;  // int: lo plane, same shape
  const void* bias;      // fp16 path: float[N]; int path: int32 correction[N]
  int K;
  int N;
  int P;                 // output pixels
  const void* src0;
  const void* src1;
  int C0, C1;
  int w8;                // width of the 1/8-scale grid
  int H, W;              // frame size
  int Csrc;              // channels of the LD_DOWN source
  void* dst;
  int Cdst;
  // prior head (EP_PRIOR*): dst = yhat_t (NHWC, Cdst = C)
  const void* y;        // NHWC latent to quantise (encode)
  const int16_t* q_in;  // planar symbols (decode)
  int16_t* q_out;       // planar symbols (encode)
  double* partials;     // one per (tile, pass) of the encoder
  const float* sigma_tab;
  uint8_t* k_out;          // planar scale indices of the entropy coder (nullable for EP_PRIOR)
  const float* scales;     // fp16 path: the NS coder scales sigma_j (fp32)
  const uint8_t* k_tab;    // int path: scale index for s_i + 32768
  // two-step entropy model
  int ld0;                 // LD_NHWC: row stride of src0 in elements (0: C0)
  int c_off;               // prior epilogues: channel of the first row pair
  const void* add;         // prior epilogues: (mu, s) added before use, NHWC; nullable
  int add_ld, add_s, add_c0;  // its row stride, offset of s, channel subtracted
  int add_f32;             // fp16 path: add is fp32 (else fp16); int path: int16
  int split;               // prior epilogues: channels >= split write (mu, s) to base (0: none)
  void* base;              // [P][2 (C - split)]: mu then s of those channels
  const float* zsigma;     // EP_ZQUANT: scale of each z channel
  const void* res;         // EP_RESID: the residual, NHWC with Cdst channels
  const uint8_t* sig8;     // EP_GATE, int path: the compact sigmoid table
  // EP_UP: workgroup 0 first sums sum_base[0, n_sum) (the rate partials of
  // the frame, written by the launches before) into *bits_out; NULL: no total
  double* bits_out;
  const double* sum_base;
  int n_sum;
};

struct BlockArgs {
  const void* w1;
  const void* w1lo;
  const void* b1;
  const void* w2;
  const void* w2lo;
  const void* b2;
  const void* dww;  // [9][C]
  const void* dwb;  // [C]
  const void* src;   // z (NHWC)
  void* dst;         // z' (NHWC), must not alias src
  int h, w;
  const void* zpad;  // C zero elements: the depthwise taps outside the image read these
  const void* sig8 = nullptr;  // int path, gated form: compact sigmoid table (896 bytes)
};

// A run of DC blocks in one launch (the C = 256 chain kernels):
// blk[b].src = blk[b - 1].dst; flags: one int per tile, zero at workspace
// creation and left equal across tiles by every launch; status: set to 1 if a
// wait for a neighbouring tile timed out.
constexpr int kMaxChain = 16;
struct DcChainArgs {
  BlockArgs blk[kMaxChain];
  int nb;
  int* flags;
  int* status;
  // fp16 chain only: when down_w is set, the last block's output stays in LDS
  // and feeds the 2x2 stride-2 downsample of the tile instead (down_w: its
  // weight fragments, K = 4C, N = C; down_b: C fp32 biases; down_y: the 1/16
  // output, NHWC), the same arithmetic as the downsample launch
  const void* down_w;
  const void* down_b;
  void* down_y;
};

struct PriorArgs {
  const void* wfrag;
  const void* wfrag_lo;
  const void* bias;       // [2C] (rows mu then s)
  const void* yhat_prev;  // NHWC latent
  const void* y;          // NHWC latent (encode)
  const int16_t* q_in;    // planar (decode)
  int16_t* q_out;         // planar (encode)
  void* yhat_new;         // NHWC latent
  double* partials;       // one per (tile, channel slice) (encode)
  const float* sigma_tab; // int path: sigma for s_i + 32768
  uint8_t* k_out;         // planar scale indices (nullable; required when scales_only)
  void* mu_out;           // scale indices only: mu (NHWC; fp32 on the fp16 path, int16 on the int path), nullable
  const float* scales;    // fp16 path: coder scales
  const uint8_t* k_tab;   // int path: scale index for s_i + 32768
  int C;
  int P;
  int decode;             // 0 encode, 1 decode (q given), 2 scale indices only
  // two-step entropy model (PwArgs fields of the same names); a step-2 call
  // has the second-step head as weights (K = C / 2, N = C) and yhat^1
  // (stride ld0) as input
  int K, N;               // 0: K = C, N = 2 C
  int ld0, c_off;
  const void* add;
  int add_ld, add_s, add_c0, add_f32;
  int split;
  void* base;
};

// Entropy coder (container and stream geometry; the tables live in the
// weights image).
constexpr int kRansStream = 8192;  // symbols per stream: 64 lanes x 128 steps
constexpr int kRansHeader = 20;    // magic, version, symbols, symbols per stream, streams
constexpr uint32_t kRansMagic = 0x5352434Eu;  // "NCRS"
constexpr uint32_t kRansVersion = 1;
constexpr int64_t kRansMaxWords = 128 + 2 * (int64_t)kRansStream;  // worst case per stream
__host__ __device__ constexpr int rans_payload_offset(int ns) { return kRansHeader + 4 * ((ns + 1) / 2); }

// Coder tables: one block of uint16 in the weights image (16-byte aligned),
// staged whole into LDS by the coder kernels.
//   [4 j .. 4 j + 3]     scale j: R_j, index of its first start, T_j and U_j,
//                        the numbers of leading and trailing entries of
//                        frequency 1 (entry i < T_j covers slot i alone, the
//                        last U_j entries the last U_j slots)
//   [256, 256 + STARTS)  starts: per scale the 2 R_j + 2 entry starts
//                        (q = -R .. R, then the escape) and a closing 0
//                        (standing for 2^16), so f_i = (start_{i+1} - start_i) mod 2^16
//   then [NS][257]       buckets: entry holding slot max(256 b, T_j) (b < 256);
//                        [256] = last entry
constexpr int kCoderStarts = 36976;  // sum over j of 2 R_j + 3
constexpr int kTabStarts = 4 * kCoderScales;
constexpr int kTabBuckets = kTabStarts + kCoderStarts;
constexpr int kTabEncU16 = kTabBuckets;                       // what the encoder stages
constexpr int kTabU16 = kTabBuckets + kCoderScales * 257;     // what the decoder stages
static_assert(kTabEncU16 % 8 == 0 && kTabU16 % 8 == 0, "coder table block must be whole 16-byte chunks");

hipError_t launch_rans_encode(const int16_t* q, const uint8_t* k, int64_t n, const uint16_t* tab, uint16_t* scratch,
                              int64_t max_words, uint32_t* lens, uint8_t* out, uint64_t* nbytes, hipStream_t st);
// errs: one word per stream; count: a zero-initialised ticket counter, left at zero
hipError_t launch_rans_decode(const uint8_t* in, uint64_t in_bytes, const uint8_t* k, int64_t n, const uint16_t* tab,
                              uint32_t* errs, uint32_t* count, int16_t* q, int32_t* status_out, hipStream_t st);

hipError_t launch_pw_f16(int loader, int epi, const PwArgs& a, hipStream_t st);
hipError_t launch_pw_i16(int loader, int epi, const PwArgs& a, hipStream_t st);
hipError_t launch_dcblock_f16(int C, bool gated, const BlockArgs& a, hipStream_t st);
hipError_t launch_dcblock128_f16(bool gated, const BlockArgs& a, hipStream_t st);  // C = 256
hipError_t launch_dcchain128_f16(bool gated, const DcChainArgs& ca, hipStream_t st);  // C = 256, fp16
int dcchain128_resident(bool gated);
// int path, LeakyReLU form, C = 256: 128 pixels per wave (one block, or a chain)
hipError_t launch_dcblock128_i16(const BlockArgs& a, hipStream_t st);
hipError_t launch_dcchain128_i16(const DcChainArgs& ca, hipStream_t st);
int dcchain128_i16_resident();
hipError_t launch_dcblock_i16(int C, bool gated, const BlockArgs& a, hipStream_t st);
hipError_t launch_prior_f16(const PriorArgs& a, hipStream_t st, int* n_partials);
hipError_t launch_prior_i16(const PriorArgs& a, hipStream_t st, int* n_partials);
int prior_partials_f16(int C, int P);
int prior_partials_i16(int C, int P);

hipError_t launch_reduce(const double* partials, int n, double* out, hipStream_t st);
constexpr int kBitsBlocks = 1024;
// sigma_tab == nullptr: scale is float32 sigma; else scale is int16 s and
// sigma = sigma_tab[s + 32768].  partials: kBitsBlocks doubles of scratch.
hipError_t launch_estimate_bits(const int16_t* q, const void* scale, const float* sigma_tab, int64_t n,
                                double* partials, double* out, hipStream_t st);
hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t st);
// yhat (NHWC, C channels, P pixels) = q (planar int16) + mu (NHWC): fp16 path
// (f16)(q + mu) with fp32 mu, int path clip(512 q + mu_i) with int16 mu_i --
// the same operations as the quantiser of the prior epilogue.
hipError_t launch_yhat_from_q(const int16_t* q, const void* mu, void* yhat, int C, int P, bool is_int,
                              hipStream_t st, int ld = 0, int c_off = 0);
// z quantiser and hyper latent (EP_ZQUANT) on the 1/16 latent y: z = W y' + b
// (y' the 2 x 2 gather), q_z planar, zhat NHWC, one rate partial per tile
hipError_t launch_zquant_f16(const PwArgs& a, hipStream_t st, int* n_partials);
hipError_t launch_zquant_i16(const PwArgs& a, hipStream_t st, int* n_partials);
// Depthwise 3x3 (zero padding) + bias of a DC block on an h x w NHWC map of
// C channels (C % 8 == 0), weights in the block's packed depthwise layout
// (fp16: per channel pair 9 tap pairs, 2 fp32 biases, a pad word; int: per
// channel quad 9 x 2 tap pairs, 4 biases 512 b, 2 pad words).  fp16: fp32
// accumulation from the bias, taps row by row, one rounding to fp16; int:
// int32 sum rescaled as every other convolution of the integer path.
hipError_t launch_dw3x3_f16(const void* src, const void* dww, void* dst, int C, int h, int w, hipStream_t st);
hipError_t launch_dw3x3_i16(const void* src, const void* dww, void* dst, int C, int h, int w, hipStream_t st);
hipError_t launch_nhwc_to_planar(const void* src, void* dst, int C, int P, hipStream_t st);
hipError_t launch_planar_to_nhwc(const void* src, void* dst, int C, int P, hipStream_t st);

// DC-block kernels tile the 1/8-scale grid in 8 x 16 pixel tiles.
inline int dc_grid(int h, int w) {
  const int t = ((h + 7) / 8) * ((w + 15) / 16);
  return (t + 7) / 8 * 8;
}

inline int grid_tiles(int P) {
  const int t = (P + 127) / 128;
  return (t + 7) / 8 * 8;
}

}  // namespace nc
