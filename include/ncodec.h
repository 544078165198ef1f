/*
 * ncodec -- C ABI of the MI355X (gfx950) implementation of the per-frame
 * transform of DCVC-RT (Jia et al., "Towards Practical Real-Time Neural Video
 * Compression", CVPR 2025).
 *
 * Problem statement followed (Sec. 4.1, Fig. 4; Sec. 5.1 "Test Details"):
 * low-delay P-frame coding.  The encoder codes frame x_t conditioned on the
 * temporal context it shares with the decoder (the previous decoded 1/8-scale
 * feature f_{t-1}, Sec. 4.3) and on the previous quantised latent; the
 * decoder, holding the same state, reproduces the frame from the symbols.
 * Encoder and decoder are separate contexts, each carrying its own state.
 *
 * Transform (one frame, C channels, h = H/8, w = W/8):
 *   patch embed     e  = W_pe * unshuffle8(x) + b_pe            (Sec. 4.2)
 *   temporal fuse   z  = W_fe * [e ; f_{t-1}] + b_fe            (Sec. 4.3)
 *   N_e DC blocks   z += W2 * LReLU_0.1(W1 * dw3x3(z) + b1) + b2 (Supp. B.1)
 *   downsample      y  = conv2x2/s2(z)                          (1/16 latent)
 *   prior           [mu ; s] = W_h * yhat_{t-1} + b_h
 *   quantise        q  = round(y - mu), yhat = q + mu           (Fig. 4 "Q")
 *   rate            bits = sum -log2 L(q; sigma), sigma = max(softplus(s), 0.11)
 *   decoder         d  = shuffle2(W_u * yhat + b_u); z' = W_fd * [d ; f_{t-1}] + b_fd;
 *                   N_d DC blocks -> f_t (the next frame's context, taken
 *                   before reconstruction, Supp. B.3)
 *   reconstruction  xhat = clamp(shuffle8(W_r * f_t + b_r), 0, 1)  (decode only)
 *
 * Integerised path (Sec. 4.5, Eq. 3; Supp. B.4, Alg. 1): features are int16
 * at K1 = 512 (1.0 -> 512), weights and biases int16 at K2 = 8192, every conv
 * accumulates conv(x_i, w_i) + 512 b_i in int32 and returns
 * clip(round_half_even(a / 8192), int16).  Results are bit-exact and
 * identical on every device.
 *
 * Conventions
 *  - Every device pointer is caller-owned device memory (e.g. a torch tensor's
 *    data_ptr()).  The library never allocates device memory: all persistent
 *    state and weights live in the caller's workspace.
 *  - Every call enqueues work on the context's HIP stream and returns without
 *    synchronising; results are valid once the stream has been synchronised.
 *  - Arguments are validated on the host before anything is enqueued.  A
 *    negative ncodec_status is returned on error; nothing is thrown across the
 *    ABI.  ncodec_last_error() gives a message.  A context is not thread-safe.
 *  - Public tensors are planar (NCHW with N = 1).  Internal layouts are
 *    private.
 */
#ifndef NCODEC_H
#define NCODEC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ncodec_ctx ncodec_ctx;

typedef enum {
  NCODEC_OK = 0,
  NCODEC_EINVAL = -1,     /* null pointer, bad enum, bad weight value        */
  NCODEC_ESHAPE = -2,     /* H, W not multiples of 16, bad C or block count   */
  NCODEC_EHIP = -3,       /* a HIP runtime call failed                        */
  NCODEC_ESTATE = -4,     /* call does not match the context's configuration  */
  NCODEC_EOVERFLOW = -5,  /* reserved: int32 accumulator overflow detected    */
  NCODEC_ENOMEM = -6      /* workspace smaller than ncodec_workspace_bytes()  */
} ncodec_status;

typedef enum { NCODEC_PATH_FP16 = 0, NCODEC_PATH_INT16 = 1 } ncodec_path;

/* Form of the DC block (Supp. B.1).  LRELU: z + pw2(LeakyReLU_0.1(pw1(dw(z))))
 * with pw2 2C -> C.  GATED: h = pw1(dw(z)) is chunked on channels into
 * (h1, h2) and the block returns z + pw2(WSiLU(h1) * h2), WSiLU(x) =
 * x sigmoid(4x), pw2 C -> C; on the int path the sigmoid is the int16 table
 * S[v] = round(512 sigmoid(4 v / 512)) (Sec. 4.5), WSiLU_i = round(h1 S[h1] / 512)
 * and the gate clip(round(WSiLU_i h2 / 512)). */
typedef enum { NCODEC_BLOCK_LRELU = 0, NCODEC_BLOCK_GATED = 1 } ncodec_block;

typedef struct {
  int32_t height;        /* H, multiple of 16, 16..8192 (caller pads 1080 -> 1088) */
  int32_t width;         /* W, multiple of 16, 16..8192                             */
  int32_t channels;      /* C in {64, 128, 256, 384, 512}; above 256 (the widths of
                            a Large model, Supp. "Performance for a Large Model")
                            each DC block runs as three launches (depthwise, pw
                            C -> 2C + LeakyReLU or the WSiLU gate, pw to C +
                            residual), in either block form                         */
  int32_t n_enc_blocks;  /* N_e, 0..32                                              */
  int32_t n_dec_blocks;  /* N_d, 0..32                                              */
  int32_t path;          /* ncodec_path                                             */
  int32_t block;         /* ncodec_block (0 = LRELU)                                */
  int32_t n_fe_blocks;   /* N_f, 0..32: feature extractor (Fig. 4; Sec. 4.3): DC
                            blocks on f_{t-1}, whose output replaces f_{t-1} as the
                            temporal context in both fuse convs                     */
  int32_t n_rg_blocks;   /* N_r, 0..32: reconstruction generation: DC blocks on f_t
                            before the reconstruction conv (decode only)            */
  int32_t qp_banks;      /* 1: the weights end with the vector banks (Sec. 4.4), see
                            ncodec_set_qp; 0: none                                  */
  int32_t hyperprior;    /* 1: the two-step entropy model with the hyper latent z
                            (Sec. 4.4; supplementary "Entropy model"), see below;
                            needs C >= 128 and H, W multiples of 32.
                            0: the one-step prior on yhat_{t-1}                     */
} ncodec_config;

/* The two-step entropy model (hyperprior = 1).  The paper codes a hyper
 * latent z with a bank of factorized modules (one per rate point; the nearest
 * one between points, Sec. 4.4 and the supplementary rate adjustment) and
 * estimates y's distribution in two steps, decoding z, then y^1, then y^2
 * (supplementary "Entropy model" and "Parallel Coding").  This library reads
 * it as:
 *   z      = conv2x2/s2(y) + b            (CZ = 64 channels at H/32 x W/32)
 *   q_z    = round(z)  (int: round(z_i / 512)), zhat = q_z (int: clip(512 q_z)),
 *            coded under a zero-mean Gaussian of scale max(zbank[qp'][c], 0.11)
 *            per channel c, qp' the nearest rate point
 *   [mu_h ; s_h] = shuffle2(W_zs zhat + b)  (2C channels at 1/16)
 *   [mu ; s] = prior(yhat_{t-1}) + [mu_h ; s_h]  (int: saturating)
 *   y^1 = channels 0 .. C/2-1, quantised with (mu, s) of those channels
 *   [dmu ; ds] = W_2 yhat^1 + b  (C/2 -> C)
 *   y^2 = channels C/2 .. C-1, quantised with mu + dmu, s + ds
 *   bits = bits(z) + bits(y^1) + bits(y^2)
 * The frame's symbols (d_q of encode / decode) are then the C x H/16 x W/16
 * planar y symbols followed by the CZ x H/32 x W/32 planar z symbols
 * (ncodec_symbol_count values).  Weights: after the vector banks, zana
 * W(CZ,C,2,2) b(CZ); zsyn W(8C,CZ) b(8C), row 4m+2i+j -> pixel-shuffle
 * position (m,i,j) of the 2C channels [mu_h ; s_h]; step2 W(C,C/2) b(C),
 * rows [dmu ; ds]; zbank (64, CZ). */

/* Number of float32 values in the canonical parameter list for cfg, or 0 if
 * cfg is invalid.  Canonical order (each weight row-major, followed by its
 * bias): pe W(C,192) b(C); fuse_enc W(C,2C) b(C) with input channels
 * [e ; f_prev]; N_e blocks of {dw W(C,3,3) b(C); pw1 W(2C,C) b(2C);
 * pw2 W(C,2C) b(C), or W(C,C) b(C) for the GATED block, whose pw1 rows are
 * [h1 ; h2]}; down W(C,C,2,2) b(C); head W(2C,C) b(2C) with rows
 * [mu ; s]; up W(4C,C) b(4C), row 4c+2i+j -> pixel-shuffle position (c,i,j);
 * fuse_dec W(C,2C) b(C) with input channels [d ; f_prev]; N_d blocks;
 * rec W(192,C) b(192), row 64c+8i+j -> colour c at pixel (8y+i, 8x+j);
 * then N_f feature-extractor blocks and N_r reconstruction-generation blocks
 * (each as the encoder's blocks); then, with qp_banks, the four vector banks
 * q_e, q_d, q_f, q_r, each 64 x C (row = rate point qp).
 * Pure host function. */
size_t ncodec_weight_count(const ncodec_config* cfg);

/* Bytes of device workspace a context needs (weights in kernel-ready form,
 * state, intermediates), or 0 if cfg is invalid.  Pure host function. */
size_t ncodec_workspace_bytes(const ncodec_config* cfg);

/* int16 symbols of one frame: C (H/16) (W/16), plus 64 (H/32) (W/32) with
 * the two-step entropy model.  0 if cfg is invalid.  Pure host function. */
size_t ncodec_symbol_count(const ncodec_config* cfg);

/* Create a context: the state of one encoder or one decoder of the low-delay
 * P-frame setting (Sec. 4.1, Fig. 4; Sec. 5.1 "Test Details"), holding the
 * weights of Fig. 4's transform and the temporal state (f_{t-1}, yhat_{t-1}),
 * Sec. 4.3.  host_weights: n_weights float32 values in canonical
 * order (host memory, copied; the fp16 path rounds them to fp16, the int
 * path converts them to round(8192 w) and rejects any weight of the
 * pointwise / 2x2 convolutions whose integer value exceeds 32639 in magnitude
 * with NCODEC_EINVAL).  d_workspace: caller-owned device buffer of at least
 * ncodec_workspace_bytes(cfg) bytes, 256-byte aligned, that must outlive the
 * context.  hip_stream: a hipStream_t (NULL = default stream).  The weight
 * upload is synchronous on that stream.  State starts as an I-frame (zero).
 * Errors: EINVAL (null pointer, wrong n_weights, weight out of range),
 * ESHAPE (bad cfg), ENOMEM (workspace too small or misaligned), EHIP. */
ncodec_status ncodec_create(const ncodec_config* cfg, const float* host_weights, size_t n_weights,
                            void* d_workspace, size_t ws_bytes, void* hip_stream, ncodec_ctx** out);

/* Make the next frame an I-frame: zero f_{t-1} and yhat_{t-1} (enqueued), so
 * the frame is coded without temporal context.  The paper's low-delay tests
 * (Sec. 5.1 "Test Details") use an intra period of -1: one I-frame starts the
 * sequence and every later frame is a P-frame, which is what a context does
 * from creation until the next reset.  Errors: EINVAL (NULL ctx), EHIP. */
ncodec_status ncodec_reset(ncodec_ctx* ctx);

/* Select rate point qp in [0, 64) of the vector banks (Sec. 4.4; the context
 * starts at qp 0).  Row qp scales per channel the latent y (q_e), the decoder
 * input yhat (q_d), the temporal context (q_f) and the generated feature
 * before the reconstruction conv (q_r); the scales are folded into the
 * adjacent convolutions (down rows, up columns, the fuse convs' context
 * columns, rec columns), each folded weight rounded to fp16, and the weights
 * are re-uploaded.  Synchronises the context's stream; the state is kept
 * (encoder and decoder must switch at the same frame).  EINVAL if the context
 * has no banks, qp is out of range, or (int path) a folded weight exceeds the
 * integer range. */
ncodec_status ncodec_set_qp(ncodec_ctx* ctx, int32_t qp);

/* Select a rate between the rate points (supplementary material, rate
 * adjustment: linear interpolation in the bank for rates between two learned
 * points).  qp is a real number in [0, 63]; with i = min(floor(qp), 62) and
 * t = qp - i, each bank vector is (1 - t) row i + t row i+1, computed in
 * double, then folded as in ncodec_set_qp.  An integer qp gives exactly row
 * qp (ncodec_set_qp(ctx, q) is ncodec_set_rate(ctx, q)).  Same
 * synchronisation, state and error behaviour as ncodec_set_qp; EINVAL for qp
 * outside [0, 63] or NaN. */
ncodec_status ncodec_set_rate(ncodec_ctx* ctx, double qp);

/* Encode one frame (Sec. 4.1, Fig. 4 encoder side, Supp. B.3 encoding).
 *  d_frame: 3 x H x W planar fp16 (IEEE binary16), values in [0, 1]; the int
 *           path converts it with x_i = round(512 x) (Alg. 1).
 *  d_q:     C x H/16 x W/16 planar int16 output symbols q (with the
 *           two-step model followed by the z symbols: ncodec_symbol_count).
 *  d_bits:  device double receiving the frame's estimated bits, or NULL.
 * Updates the context state to (f_t, yhat_t).  d_frame must not alias d_q. */
ncodec_status ncodec_encode_frame(ncodec_ctx* ctx, const void* d_frame, int16_t* d_q, double* d_bits);

/* Decode one frame from its symbols (Fig. 4 decoder side, Supp. B.3).
 *  d_q:         the symbols from ncodec_encode_frame (ncodec_symbol_count).
 *  d_frame_out: 3 x H x W planar; fp16 in [0,1] (fp16 path) or int16 in
 *               [0, 512] (int path).
 * Updates the context state to (f_t, yhat_t). */
ncodec_status ncodec_decode_frame(ncodec_ctx* ctx, const int16_t* d_q, void* d_frame_out);

/* Rate of n symbols under zero-mean Gaussians (Supp. B.2; likelihood
 * L = Phi((|q|+1/2)/sigma) - Phi((|q|-1/2)/sigma), bits = sum -log2 max(L, 1e-9)).
 *  d_q:     n int16 symbols.
 *  d_scale: n scales in the form the context's path produces them: on an
 *           fp16 context float32 sigma (> 0); on an int16 context the prior's
 *           int16 scale outputs s_i (K1 = 512 units), each mapped to
 *           sigma = max(softplus(s_i / 512), 0.11) through the context's table
 *           of all 65,536 values (Sec. 4.5: table lookups keep the integer path
 *           identical across devices).
 *  d_bits:  device double output.
 * The sum is formed in a fixed order (deterministic).  n must be in
 * [0, 2^31); n = 0 writes 0.  Uses the context's workspace as scratch, so
 * calls on one context are ordered by its stream. */
ncodec_status ncodec_estimate_bits(ncodec_ctx* ctx, const int16_t* d_q, const void* d_scale,
                                   int64_t n, double* d_bits);

/* ncodec_estimate_bits without a context, for callers that cannot allocate
 * device memory (code under graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Same rate, same fixed summation order and the same
 * result bit for bit as ncodec_estimate_bits on an fp16 context: d_q n int16
 * symbols, d_sigma n float32 scales, *d_bits (device double) the total.
 * Enqueued on hip_stream (a hipStream_t; NULL = default stream) on the
 * current device.  Allocates nothing: its partial sums live in a static
 * device array of 1,024 doubles (8 KiB) that each GPU the library runs on
 * holds until the process ends.  All calls on one GPU share that array, so
 * calls that overlap on one GPU (different streams, or threads without
 * ordering) race; calls ordered on one stream do not.  n must be in
 * [0, 2^31) (any n uses the same 1,024 partials); NCODEC_EINVAL otherwise or
 * for a NULL d_bits (or NULL d_q / d_sigma with n > 0), NCODEC_EHIP for a
 * HIP failure; ncodec_last_error(NULL) gives the message. */
ncodec_status ncodec_estimate_bits_noalloc(const int16_t* d_q, const float* d_sigma, int64_t n,
                                           double* d_bits, void* hip_stream);

/* ---- Entropy coding (Fig. 4 "AE" / "AD", Fig. 6; Supp. B.2) ----------------
 * The symbols are coded with rANS (Duda 2013; 32-bit state in [2^16, 2^32),
 * 16-bit words, 16-bit frequencies) under quantised-scale Gaussian tables:
 * NS = 64 scales sigma_j = fp32(0.11 (256/0.11)^(j/63)); table j codes
 * q = -R .. R (R = max(ceil(8 sigma_j), 32)) and an escape for larger |q|,
 * which is followed by one 16-bit field of frequency 1,
 * 32768 * sign + |q| - R - 1.  Frequencies: f = 1 + floor(p (2^16 - n)) for each of the
 * n = 2R + 2 symbols of the Gaussian of scale sigma_j, the remainder added at
 * q = 0.  The scale index of a symbol is the smallest j with
 * sigma_j >= sigma = max(softplus(s), 0.11) (s the prior's scale output; on the
 * int path s is an int16 and the index comes from a table of all 65,536
 * values, so encoder and decoder agree on any device, Sec. 4.5).
 *
 * Container (little-endian bytes): u32 magic "NCRS", u32 version 1, u32 number
 * of symbols, u32 symbols per stream (8192), u32 number of streams, u16 length
 * in words of each stream, zero padding to 4 bytes, then the streams' 16-bit
 * words.  A stream's 8192 symbols are coded by 64 interleaved rANS states
 * (symbol i by state i % 64); it opens with the 64 final states.
 *
 * All calls enqueue on the context's stream; byte counts and status words are
 * device outputs, valid after the stream synchronises.  Buffers must be device
 * memory; d_stream must be 4-byte aligned, symbol and scale-index arrays
 * 16-byte aligned.  A stream holds at most 128 + 2 * 8192 words. */

/* Worst-case container size in bytes for one frame of cfg (what d_stream
 * must hold for ncodec_encode_frame_coded).  0 for an invalid cfg.  With the
 * two-step entropy model a frame is three containers, z, y^1 and y^2, each
 * at a fixed offset: 0, cap(nz), cap(nz) + cap(n1), with cap(n) the
 * worst case of n symbols (nz = 64 (H/32) (W/32), n1 = n2 = C/2 (H/16) (W/16)),
 * and the capacity is their sum. */
size_t ncodec_stream_capacity(const ncodec_config* cfg);

/* Scale indices (uint8, C x H/16 x W/16 planar) of the symbols of the next
 * frame, from the current state (the prior head on yhat_{t-1}).  ESTATE with
 * the two-step model (its indices depend on the frame's z and y^1). */
ncodec_status ncodec_scale_indices(ncodec_ctx* ctx, uint8_t* d_k);

/* Code n symbols d_q (int16) with scale indices d_k (uint8, values >= 64 are
 * taken as 63) into the container d_stream (capacity bytes, at least the
 * worst case for n symbols: ncodec_stream_capacity of a frame with n symbols).
 * *d_stream_bytes (device u64) receives the container size.
 * n must be in [1, C H W / 256] of the context's frame.  EINVAL otherwise. */
ncodec_status ncodec_rans_encode(ncodec_ctx* ctx, const int16_t* d_q, const uint8_t* d_k, int64_t n,
                                 void* d_stream, size_t capacity, uint64_t* d_stream_bytes);

/* Decode n symbols from a container of stream_bytes bytes with scale indices
 * d_k into d_q.  *d_status (device int32, may be NULL) receives 0 for a clean
 * decode, else a bit set: 1 bad or truncated container, 2 a stream ran past
 * its length, 4 a stream ended in an inconsistent state.  The decoder never
 * reads outside [d_stream, d_stream + stream_bytes); on error the symbols are
 * unspecified but written in full. */
ncodec_status ncodec_rans_decode(ncodec_ctx* ctx, const void* d_stream, size_t stream_bytes, const uint8_t* d_k,
                                 int64_t n, int16_t* d_q, int32_t* d_status);

/* ncodec_encode_frame, then the frame's symbols coded into d_stream
 * (capacity >= ncodec_stream_capacity(cfg)); *d_stream_bytes (device u64)
 * receives the container size (two-step model: d_stream_bytes[0 .. 2], the
 * sizes of the z, y^1 and y^2 containers).  d_q (symbols) and d_bits
 * (estimate) may be NULL. */
ncodec_status ncodec_encode_frame_coded(ncodec_ctx* ctx, const void* d_frame, int16_t* d_q, double* d_bits,
                                        void* d_stream, size_t capacity, uint64_t* d_stream_bytes);

/* Decode one frame from its container: scale indices from the state, symbols
 * from the container, then ncodec_decode_frame.  *d_status as for
 * ncodec_rans_decode (may be NULL; two-step model: d_status[0 .. 2] for the
 * z, y^1 and y^2 containers, decoded in that order, each with the
 * distribution that the previous ones determine); the state advances even on
 * error.  stream_bytes bounds every read. */
ncodec_status ncodec_decode_frame_coded(ncodec_ctx* ctx, const void* d_stream, size_t stream_bytes,
                                        void* d_frame_out, int32_t* d_status);

/* Parallel coding (Fig. 6; supplementary "Parallel Coding"): with enable != 0
 * the coded calls overlap entropy coding with the network parts that do not
 * depend on it.  ncodec_encode_frame_coded runs the rANS coder on a second
 * HIP stream (default priority, created on first use) as soon as the symbols
 * and their scale indices exist, while the decoder part of the encode runs on
 * the context's stream; ncodec_decode_frame_coded runs the feature extractor
 * (n_fe_blocks > 0) on the second stream while the symbols are decoded.  Both
 * join the context's stream with an event before its last launches, so
 * results are valid, as always, once the context's stream has synchronised,
 * and are identical to the serial order (the default, enable = 0). */
ncodec_status ncodec_parallel_coding(ncodec_ctx* ctx, int32_t enable);

/* Copy the state out of / into the context (enqueued): the temporal context
 * f_{t-1} (the decoder feature before reconstruction, Sec. 4.3; Supp. B.3) and
 * the previous latent yhat_{t-1} that the prior reads.  Encoder and decoder
 * hold the same state after every frame (Sec. 4.5: on the int path bitwise,
 * on any device), so a state copied from one context continues the stream in
 * another.  d_feat: C x H/8 x W/8 planar, d_yhat: C x H/16 x W/16 planar; fp16
 * (fp16 path) or int16 (int path), caller-owned device memory, 16-byte
 * aligned.  Either pointer may be NULL to skip that tensor.  Errors: EINVAL
 * (NULL ctx), EHIP. */
ncodec_status ncodec_get_state(ncodec_ctx* ctx, void* d_feat, void* d_yhat);
ncodec_status ncodec_set_state(ncodec_ctx* ctx, const void* d_feat, const void* d_yhat);

/* Kernel launches one ncodec_encode_frame (decode = 0; one workgroup of the
 * upsample that follows the prior sums the frame's bit total, so d_bits does
 * not change the count) or ncodec_decode_frame (decode = 1) enqueues (three more each with
 * the two-step model; on the fp16 path the upsample and its fuse conv are one
 * launch, and so are the patch embed and its fuse conv; a chain of DC blocks
 * counts as one launch per up to 16 blocks, see ncodec_block_chains, and on
 * the fp16 path the encoder's last chain also runs the downsample),
 * counting the feature-extractor and reconstruction-generation blocks
 * (Sec. 3: the number of modules called per frame is one of the costs the
 * design minimises).  0 for a NULL ctx. */
int32_t ncodec_kernels_per_frame(const ncodec_ctx* ctx, int32_t decode);

/* Graph replay of the per-frame launch sequence (Sec. 3: at this size the
 * module count, not the MAC count, is what costs time).  When enabled, the
 * first encode (decode) for each of the two state buffers captures its
 * launches into a hipGraph on a private stream; later calls replay it on the
 * context's stream, re-pointing only the nodes that read or write the
 * caller's buffers (frame, q, bits, output frame).  Results are identical to
 * the direct launches.  Off by default: on MI355X with ROCm 7 the replay of
 * this linear launch chain measured slightly slower than direct launches.
 * While per-kernel timing is enabled, calls launch directly.  Errors: EHIP if
 * capture, instantiation, update or launch fails. */
ncodec_status ncodec_graph_enable(ncodec_ctx* ctx, int32_t enable);

/* Block chains (Sec. 3: fewer, larger modules per frame; Supp. B.1 blocks run
 * back to back).  At C = 256 (fp16 path, either block form; int16 path, the
 * LeakyReLU form) the consecutive DC blocks of a
 * transform (the encoder's, the decoder's, the feature extractor's, the
 * reconstruction generation's; up to 16 per launch) run as one launch (on the
 * fp16 path the encoder's together with the downsample) in which
 * every 8 x 16 tile keeps its block output on chip and exchanges only its edge
 * pixels with the neighbouring tiles through memory.  Used only where every
 * tile fits the device at once (checked once per context with the occupancy
 * API; 255 tiles of one workgroup per CU at 1080p); otherwise, and with
 * enable = 0, one launch per block.  Results are identical either way.  On by
 * default.  A tile waits at most about 0.1 s for a neighbour (a case that
 * needs another kernel holding CUs for that long); a wait that gives up
 * leaves the block outputs wrong and is reported by
 * ncodec_block_chain_status.  Changing the setting drops captured graphs (the
 * next graph call captures again).  Errors: EINVAL for a NULL ctx, EHIP. */
ncodec_status ncodec_block_chains(ncodec_ctx* ctx, int32_t enable);

/* *in_use = 1 if this context's DC blocks run as chains (enabled, fp16,
 * C = 256 and every tile resident at once), else 0.  Synchronizes the
 * context's stream and writes to *timeouts 1 if any chain launch of this
 * context has given up waiting for a neighbouring tile since its creation,
 * else 0.  Errors: EINVAL for a NULL ctx, in_use or timeouts, EHIP. */
ncodec_status ncodec_block_chain_status(ncodec_ctx* ctx, int32_t* in_use, int32_t* timeouts);

/* Optional per-kernel timing.  While enabled, the kernels the context
 * enqueues are launched with HIP events attached to their dispatch
 * (hipExtLaunchKernel): a start event on the first launch of each run of
 * consecutive launches of one kind (the DC blocks of a transform form one
 * run) and a stop event on its last, so each interval is the run's execution
 * time including the gaps inside it, and the per-launch average is that
 * interval over the run's launch count.  ncodec_timing_read() synchronises
 * the stream, aggregates the intervals per kernel kind (launch count and
 * summed milliseconds), writes at most max_kinds records to out, sets
 * *n_kinds, and clears the log.  Kinds: "embed", "fuse", "embed_fuse",
 * "dcblock" (wide blocks: "dcblock_dw", "dcblock_pw1", "dcblock_pw2"), "down",
 * "prior", "up", "up_fuse", "recon", "zquant", "hyper", "zhat", "yhat",
 * "rans_enc", "rans_dec", "dcblock_down" (the fp16 encoder's chain that also
 * runs the downsample; it has no "down" launch).  A chain of DC blocks
 * (ncodec_block_chains) counts as one launch per block, so "dcblock" is
 * always per block.  Meant for
 * measurement runs; off by default. */
typedef struct {
  char kind[16];
  int32_t launches;
  double total_ms;
} ncodec_kernel_timing;

ncodec_status ncodec_timing_enable(ncodec_ctx* ctx, int32_t enable);
ncodec_status ncodec_timing_read(ncodec_ctx* ctx, ncodec_kernel_timing* out, int32_t max_kinds, int32_t* n_kinds);

/* Message for the last error on ctx (or the last create failure if ctx is NULL). */
const char* ncodec_last_error(const ncodec_ctx* ctx);

/* Static description of a status code. */
const char* ncodec_status_string(ncodec_status st);

/* Release host resources of the context (the workspace stays caller-owned).
 * Synchronises the context's stream first.  NULL is ignored. */
void ncodec_destroy(ncodec_ctx* ctx);

#ifdef __cplusplus
}
#endif
#endif /* NCODEC_H */
