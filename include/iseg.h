/*
 * iseg.h -- C ABI of libiseg.so, the MI355X (gfx950) kernels of the integer
 * training dataflow of "Training and Inference for Integer-Based Semantic
 * Segmentation Network" (arXiv 2011.14504, Sec. 3).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Quantized tensor.  A tensor of integer codes n plus ONE int32 exponent e per
 * tensor; the value of an element is n * 2^e.  Codes of a k-bit object lie in
 * [-(2^(k-1)-1), 2^(k-1)-1] (the clip range of Eq. 2): no entry point ever
 * writes -128.  The compute entry points do not re-check their inputs (a pass
 * over every input per call would cost about as much as the call itself): an
 * input code of -128 is computed exactly as the value -128 * 2^e, and every
 * bound below allows for it.  Tensors from outside the library can be checked
 * once with iseg_check_codes.  Exponents live in DEVICE memory (one int32 each) so
 * that a producer's data-dependent scale reaches its consumer without a host
 * round trip.
 *
 * Layouts.  Activations and errors: NHWC, contiguous, int8.  Conv weights:
 * KRSC (out-channel, kernel row, kernel column, in-channel), int8 codes;
 * masters int32.  Per-channel vectors: C.
 *
 * Pointers.  Every data pointer is a device pointer unless said otherwise;
 * geometry/config structs are HOST pointers read during the call.  The caller
 * owns all memory.  The library never allocates: scratch space comes from a
 * caller workspace `ws` of at least the size returned by the matching
 * iseg_*_ws() query (256-byte aligned).  Inputs and outputs must not alias.
 * The workspaces of iseg_bn_fwd and iseg_bn_bwd begin with arrival counters
 * (ISEG_BN_WS_ZERO(C) bytes) that must be zero before the first call with
 * that buffer: zero it once when it is allocated.  Every iseg_bn_fwd /
 * iseg_bn_bwd call leaves them zero again, so a buffer kept for those calls
 * on one stream stays ready; a buffer that other entry points also use must
 * be zeroed again before the next L1BN call, and calls that may run at the
 * same time need buffers of their own.
 *
 * Streams.  Every compute call only enqueues work on `stream` (0 = the null
 * stream) and returns; results are ready when the stream reaches that point.
 *
 * Errors.  Return values are synchronous host checks: ISEG_OK, or
 * ISEG_ERR_ARG / _SHAPE / _UNSUPPORTED / _WORKSPACE before anything is
 * enqueued, or ISEG_ERR_DEVICE if a launch failed.  Conditions only the device
 * can see (an exponent outside a documented range, a non-finite float) are
 * OR-ed as ISEG_DEV_* bits into the caller's sticky int32 `dev_status` word (device
 * memory, may be NULL); outputs are then unspecified.
 *
 * Scale rule.  Scale(x) = max|x| (Eq. 3) is realized as the smallest power of
 * two strictly greater than max|x|, so every scale is an exponent shift and
 * requantizing a tensor that already holds k-bit codes is value-exact.
 * Rounding is half-up (floor(x/Delta + 1/2), Eq. 2) unless stochastic
 * (Eq. 5-6).  A tensor whose maximum is 0 gets codes 0 and keeps its input
 * exponent.
 *
 * Stochastic rounding draws come from Philox4x32-10 with key (seed mod 2^32,
 * tensor_id) and counter (idx mod 2^32, idx >> 32, step, 0), idx the element's
 * linear index in the output layout; the draw is w0 | w1 << 32 and the top r
 * bits decide a rounding of r fractional bits.
 */
#ifndef ISEG_H
#define ISEG_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

enum iseg_status {
    ISEG_OK = 0,
    ISEG_ERR_ARG = 1,          /* bad pointer, bit-width or mode */
    ISEG_ERR_SHAPE = 2,        /* inconsistent or empty-but-invalid geometry */
    ISEG_ERR_UNSUPPORTED = 3,  /* valid but outside what the kernels cover */
    ISEG_ERR_WORKSPACE = 4,    /* ws NULL or smaller than the query says */
    ISEG_ERR_DEVICE = 5        /* a HIP launch failed */
};

/* bits OR-ed into *dev_status by kernels */
enum iseg_dev_status {
    ISEG_DEV_RANGE = 1,        /* an exponent outside its documented range */
    ISEG_DEV_NONFINITE = 4,    /* a NaN or infinity in a float input */
    ISEG_DEV_DESC = 8          /* a device descriptor field out of range (entry skipped) */
};

enum iseg_dtype { ISEG_I8 = 0, ISEG_I16 = 1, ISEG_I32 = 2, ISEG_I64 = 3 };

enum iseg_qmode { ISEG_Q_UQ = 0, ISEG_Q_SQ = 1 };

/* conv output: SQ to 8 bits (int8 codes), or the raw exact int32 sums */
enum iseg_out_mode { ISEG_OUT_Q8 = 0, ISEG_OUT_RAW = 1 };

/* weight-gradient quantizer: Eq. 17 keeps Scale(G), Eq. 18 drops it; RAW
 * returns the exact int64 sums */
enum iseg_g_mode { ISEG_G_KEEP = 0, ISEG_G_DROP = 1, ISEG_G_RAW = 2 };

/* bytes of arrival counters at the head of an L1BN (iseg_bn_fwd /
 * iseg_bn_bwd) workspace for C channels */
#define ISEG_BN_WS_ZERO(C) ((((size_t)(C) + 511) / 256) * 256)

/* Convolution geometry.  Input NHWC [N,H,W,C]; weights KRSC [K,R,S,C];
 * output [N,P,Q,K] with P = floor((H + 2 pad_h - dil_h (R-1) - 1)/stride_h)+1
 * (Q likewise).  Zero padding, cross-correlation, no bias. */
typedef struct iseg_conv_geom {
    int64_t N, H, W, C;
    int64_t K, R, S;
    int32_t stride_h, stride_w, pad_h, pad_w, dil_h, dil_w;
} iseg_conv_geom;

/* L1BN bit-widths (Sec. 3.2.2, Eq. 14; defaults from Sec. 5: 16,16,16,8,8)
 * plus the activation/error widths around it and two readings the paper
 * leaves open: eps_code (epsilon in LSBs of the sigma grid) and relu (apply a
 * ReLU between the affine step and Q_A). */
typedef struct iseg_bn_cfg {
    int32_t k_mu, k_sigma, k_xhat, k_gamma, k_beta;
    int32_t k_A, k_E1, k_E2;
    int32_t eps_code, relu;
} iseg_bn_cfg;

/* ------------------------------------------------------------------------ */
/* Quantizers                                                                */
/* ------------------------------------------------------------------------ */

/* iseg_quantize -- float32 tensor to integer codes (Eq. 2 UQ, or Eq. 3-4 SQ
 * with the power-of-two Scale).  UQ: code = clamp(floor(x 2^(bits-1) + 1/2)),
 * exponent 1-bits.  SQ: b = exponent of the smallest power of two strictly
 * above max|x| (0 for an all-zero tensor), code = clamp(floor(x 2^(bits-1-b) +
 * 1/2)), exponent b+1-bits.
 *   x [n] float32 (device); bits in [2, 31]; out_dtype ISEG_I8 (bits <= 8),
 *   ISEG_I16 (bits <= 16) or ISEG_I32; out [n]; out_exp: one device int32.
 *   Non-finite input sets ISEG_DEV_NONFINITE. */
size_t iseg_quantize_ws(int64_t n);
int iseg_quantize(const float* x, int64_t n, int32_t bits, int32_t mode,
                  int32_t out_dtype, void* out, int32_t* out_exp,
                  void* ws, size_t ws_bytes, int32_t* dev_status, hipStream_t stream);

/* iseg_requant -- SQ (Eq. 4) or stochastic RQ (Eq. 5-6) of an integer tensor.
 * With M = max|in| and r = bitlen(M) - (bits-1): code = clamp(floor(in/2^r +
 * 1/2)) (half-up) or clamp(floor(in/2^r) + [u_r < in mod 2^r]) (stochastic,
 * u_r the top r bits of the element's Philox draw); for r <= 0 code =
 * in * 2^-r exactly.  Exponent in_exp + r (keep_scale = 1, Eq. 4 / Eq. 17) or
 * 1-bits (keep_scale = 0, Eq. 18).
 *   in [n] of in_dtype ISEG_I32 or ISEG_I64; in_exp device int32 (ignored
 *   when keep_scale = 0); bits in [2, 16]; out_dtype ISEG_I8 (bits <= 8) or
 *   ISEG_I16. */
size_t iseg_requant_ws(int64_t n);
int iseg_requant(const void* in, int32_t in_dtype, int64_t n, const int32_t* in_exp,
                 int32_t bits, int32_t stochastic, int32_t keep_scale,
                 uint64_t seed, uint32_t tensor_id, uint32_t step,
                 int32_t out_dtype, void* out, int32_t* out_exp,
                 void* ws, size_t ws_bytes, int32_t* dev_status, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Convolutions (int8 x int8 -> exact int32 sums on MFMA, then a quantizer)  */
/* ------------------------------------------------------------------------ */

/* iseg_conv_fwd -- y[n,p,q,k] = sum_{r,s,c} x[n, p st_h - pad_h + r dil_h,
 * q st_w - pad_w + s dil_w, c] * w[k,r,s,c]; then Q_A = SQ(., 8) (Eq. 15) for
 * ISEG_OUT_Q8 (y int8, y_exp = x_exp + w_exp + r) or the raw sums for
 * ISEG_OUT_RAW (y int32, y_exp = x_exp + w_exp).  The weights are W_q of
 * Eq. 8.  ISEG_OUT_RAW requires C*R*S <= 131071 so the exact sums fit
 * int32.  ISEG_OUT_Q8 also takes longer reductions, cut over C into at most 8
 * chunks of a multiple of 16 channels with at most 131071 products each (a
 * 7x7 conv over up to 21376 channels): every chunk's exact int32 sums are
 * kept in the workspace and the quantizer adds them in int64, so the codes
 * are those of the exact total; ISEG_ERR_UNSUPPORTED beyond that. */
size_t iseg_conv_fwd_ws(const iseg_conv_geom* g, int32_t out_mode);
int iseg_conv_fwd(const int8_t* x, const int32_t* x_exp, const int8_t* w, const int32_t* w_exp,
                  const iseg_conv_geom* g, int32_t out_mode, void* y, int32_t* y_exp,
                  void* ws, size_t ws_bytes, int32_t* dev_status, hipStream_t stream);

/* iseg_conv_bwd_data -- the adjoint of iseg_conv_fwd: dx[n,h,w,c] = sum of
 * dy[n,p,q,k] * w[k,r,s,c] over h = p st_h - pad_h + r dil_h, w = q st_w -
 * pad_w + s dil_w; then Q_E = SQ(., 8) (Eq. 16) for ISEG_OUT_Q8 (dx int8,
 * dx_exp = dy_exp + w_exp + r) or the raw int32 sums.  dy is [N,P,Q,K];
 * dx is [N,H,W,C].  ISEG_OUT_RAW requires K*R*S <= 131071; ISEG_OUT_Q8
 * splits a longer reduction over K as iseg_conv_fwd splits one over C (FCN's
 * fc6, 7x7 from 4096 channels, takes two chunks). */
size_t iseg_conv_bwd_data_ws(const iseg_conv_geom* g, int32_t out_mode);
int iseg_conv_bwd_data(const int8_t* dy, const int32_t* dy_exp, const int8_t* w, const int32_t* w_exp,
                       const iseg_conv_geom* g, int32_t out_mode, void* dx, int32_t* dx_exp,
                       void* ws, size_t ws_bytes, int32_t* dev_status, hipStream_t stream);

/* Transposed weight layouts that backward-data convolves dy with (Eq. 16's
 * adjoint): ISEG_WT_CRSK is wt[c][r][s][k] = w[k][r][s][c]; ISEG_WT_CRSK_FLIP
 * also reverses the taps, wt[c][R-1-r][S-1-s][k] (stride-1 paths). */
enum iseg_wt_kind { ISEG_WT_NONE = 0, ISEG_WT_CRSK = 1, ISEG_WT_CRSK_FLIP = 2 };

/* iseg_conv_bwd_data_wt_kind -- the layout iseg_conv_bwd_data builds in its
 * workspace for this geometry (ISEG_WT_NONE for an invalid geometry, and for
 * a reduction split over K, whose chunks read w itself). */
int32_t iseg_conv_bwd_data_wt_kind(const iseg_conv_geom* g);

/* iseg_conv_bwd_data_t -- iseg_conv_bwd_data with the transposed weights
 * supplied by the caller: wt (device, 16-byte aligned, K*R*S*C bytes) holds
 * w in layout wt_kind, e.g. from iseg_weight_transpose_multi after the last
 * weight update.  When the path chosen for the call needs another layout
 * (or wt is NULL / unaligned) it builds its own from w as iseg_conv_bwd_data
 * does, so the result is the same either way; w must always be valid.
 * ISEG_ERR_ARG for an unknown wt_kind. */
int iseg_conv_bwd_data_t(const int8_t* dy, const int32_t* dy_exp, const int8_t* w, const int32_t* w_exp,
                         const int8_t* wt, int32_t wt_kind, const iseg_conv_geom* g, int32_t out_mode,
                         void* dx, int32_t* dx_exp, void* ws, size_t ws_bytes, int32_t* dev_status,
                         hipStream_t stream);

/* One weight tensor of iseg_weight_transpose_multi: w [K][RS][C] int8 -> wt
 * in layout kind (ISEG_WT_CRSK or ISEG_WT_CRSK_FLIP, RS = R*S taps).  The
 * tensor is cut into ceil(C/64) * ceil(K/64) * RS tiles; tile_begin is the
 * number of tiles of the descriptors before it (descriptors in order). */
typedef struct iseg_wt_desc {
    const int8_t* w;
    int8_t* wt;
    int32_t K, RS, C, kind;
    int64_t tile_begin;
} iseg_wt_desc;

/* iseg_weight_transpose_multi -- every descriptor's transposed copy in one
 * launch (one 64 x 64 LDS tile per block).  descs: device array of n_desc
 * descriptors (caller-owned, outputs must not overlap); total_tiles = the
 * last tile_begin plus that descriptor's tile count.  Not part of the
 * paper's arithmetic: a data layout for the backward-data convolutions. */
int iseg_weight_transpose_multi(const iseg_wt_desc* descs, int32_t n_desc, int64_t total_tiles,
                                hipStream_t stream);

/* iseg_conv_bwd_weight -- G[k,r,s,c] = sum_{n,p,q} dy[n,p,q,k] * x[n, p st_h -
 * pad_h + r dil_h, q st_w - pad_w + s dil_w, c] exactly (int32 partial sums of
 * at most 131008 pixels, added in int64); then Q_G: stochastic RQ to `bits`
 * (Eq. 5-6) keeping the scale (ISEG_G_KEEP, Eq. 17: dw_exp = dy_exp + x_exp +
 * r) or dropping it (ISEG_G_DROP, Eq. 18: dw_exp = 1-bits); dw int8 [K,R,S,C].
 * ISEG_G_RAW writes the int64 sums (dw_exp = dy_exp + x_exp).  Philox index =
 * the KRSC linear index. */
size_t iseg_conv_bwd_weight_ws(const iseg_conv_geom* g, int32_t g_mode);
int iseg_conv_bwd_weight(const int8_t* dy, const int32_t* dy_exp, const int8_t* x, const int32_t* x_exp,
                         const iseg_conv_geom* g, int32_t g_mode, int32_t bits,
                         uint64_t seed, uint32_t tensor_id, uint32_t step,
                         void* dw, int32_t* dw_exp,
                         void* ws, size_t ws_bytes, int32_t* dev_status, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* L1 batch normalization (Eq. 12-15) and its backward                       */
/* ------------------------------------------------------------------------ */

/* iseg_bn_fwd -- per channel c of x [M, C] (M = N*H*W, codes with exponent
 * s_x in [-40, 16], M <= 2^22, C % 4 == 0):
 *   mu_q  = 2 UQ(mu/2, k_mu), mu the batch mean            (Eq. 10, 14)
 *   sigma = mean |x - mu_q|; sigma_q = 2 UQ(sigma/2, k_sigma) (Eq. 13, 14)
 *   xhat  = (x - mu_q) / (sigma_q + eps)                    (Eq. 12)
 *           with the denominator code max(n_sigma + eps_code, 1)
 *   xhat_q= SQ(xhat, k_xhat), one scale for the tensor      (Eq. 14)
 *   y     = gamma_q xhat_q + beta_q, ReLU if cfg->relu      (Eq. 12)
 *   A     = SQ(y, k_A) -> y_out int8, y_exp                 (Eq. 15)
 * gamma_q / beta_q: [C] int8 codes of Q_gamma / Q_beta (value n 2^(2-k)).
 * An all-zero xhat takes b = 0.  s_x outside its range sets ISEG_DEV_RANGE.
 * `saved` (iseg_bn_saved_bytes(C) bytes, device) receives what the backward
 * needs; its layout is:
 *   int32 hdr[16]: [0] b (xhat_q exponent is b+1-k_xhat), [1] y grid exponent,
 *                  [2] A exponent, [3] s_x;
 *   then, each 256-byte aligned: int32 n_mu[C], n_sigma[C], den[C] (the
 *   denominator code), qmin[C], qmax[C] (occupied input-code range), t0[C]
 *   (least code with x >= mu_q), p0[C] (least code with x > mu_q), mlo[C],
 *   mhi[C] (codes with y > 0 form [mlo, mhi]); int16 xhat_code[C][256] (by
 *   input code + 128); uint8 flags[C][256] (bit0: y > 0, bits1-2: sgn(x -
 *   mu_q) + 1); int8 a_code[C][256]; uint32 bwd_entry[C][256] (by the
 *   input code's byte, q & 0xff: bit0 y > 0, bits 8-9 sgn(x - mu_q) as a
 *   two-bit signed field, bit 10 |sgn|, bits 16-31 the xhat code); int16
 *   y_staged[C][256] (by input code + 128: ReLU(y) on the y grid floored by
 *   2^t_c, t_c = max(0, r_c - 1) with r_c the Q_A shift of channel c's own
 *   max |ReLU(y)|, clamped to +-32767; the output pass's working copy). */
size_t iseg_bn_saved_bytes(int64_t C);
size_t iseg_bn_fwd_ws(int64_t M, int64_t C);
int iseg_bn_fwd(const int8_t* x, const int32_t* x_exp, int64_t M, int64_t C,
                const int8_t* gamma_q, const int8_t* beta_q, const iseg_bn_cfg* cfg,
                int8_t* y_out, int32_t* y_exp, void* saved,
                void* ws, size_t ws_bytes, int32_t* dev_status, hipStream_t stream);

/* iseg_bn_fwd_noalloc -- iseg_bn_fwd for callers that cannot allocate
 * device memory (code under graph capture, serving loops, harnesses that
 * forbid hipMalloc): the same computation and outputs, with the workspace in
 * a static device array of iseg_bn_fwd_noalloc_max_bytes() bytes (1 MiB,
 * one per GPU, held until the process ends) instead of a caller buffer.
 * Enough for every C <= 32768 at any M; a shape whose iseg_bn_fwd_ws()
 * exceeds it returns ISEG_ERR_WORKSPACE before anything is enqueued.  Every
 * call on a GPU uses that GPU's one array: calls that overlap on one GPU
 * (other streams, other threads) race and must be serialized by the caller.
 * Nothing has to be cleared between calls: the array starts at zero and
 * every call leaves its arrival counters at zero.  Allocates nothing (no hipMalloc,
 * no library routine that allocates); the array's device address is looked
 * up once per device on the first call there (ISEG_ERR_DEVICE if that
 * fails). */
size_t iseg_bn_fwd_noalloc_max_bytes(void);
int iseg_bn_fwd_noalloc(const int8_t* x, const int32_t* x_exp, int64_t M, int64_t C,
                        const int8_t* gamma_q, const int8_t* beta_q, const iseg_bn_cfg* cfg,
                        int8_t* y_out, int32_t* y_exp, void* saved, int32_t* dev_status,
                        hipStream_t stream);

/* iseg_bn_bwd -- exact derivative of Eq. 12-13 with straight-through
 * quantizers (the paper prints no backward formula), for the forward that
 * filled `saved` from the same x:
 *   delta  = dy * [y > 0] (ReLU mask only if cfg->relu)
 *   dbeta  = sum delta      -> dbeta[C] int64,  *dbeta_exp  = dy_exp
 *   dgamma = sum delta xhat_q -> dgamma[C] int64, *dgamma_exp = dy_exp + exp(xhat_q)
 *   E2     = SQ(gamma_q delta, k_E2)                         (Eq. 16)
 *   dx     = [E2 - mean E2 - mean(E2 xhat_q) (s - mean s)] / (sigma_q + eps),
 *            s = sgn(x - mu_q), means over the channel's M values
 *   E1     = SQ(dx, k_E1) -> dx_out int8, dx_exp                (Eq. 16)
 * dy [M, C] int8 with exponent in [-60, 16]. */
/* workspace of iseg_bn_bwd; its first ISEG_BN_WS_ZERO(C) bytes are the
 * arrival counters described under Pointers */
size_t iseg_bn_bwd_ws(int64_t M, int64_t C);
int iseg_bn_bwd(const int8_t* dy, const int32_t* dy_exp, const int8_t* x,
                int64_t M, int64_t C, const int8_t* gamma_q, const iseg_bn_cfg* cfg,
                const void* saved, int8_t* dx_out, int32_t* dx_exp,
                int64_t* dgamma, int64_t* dbeta, int32_t* dgamma_exp, int32_t* dbeta_exp,
                void* ws, size_t ws_bytes, int32_t* dev_status, hipStream_t stream);

/* Inference with frozen statistics.  The paper claims fixed-point inference
 * (Sec. 1, 6) but gives no rule for running statistics; the reading taken:
 * a layer's inference state is the state one calibration forward in training
 * mode (iseg_bn_fwd) saved -- per channel n_mu and the denominator, and the
 * exponents of its input Z, of Q_xhat (b) and of Q_A -- and later inputs use
 * it unchanged: every quantizer keeps the calibration's step and clips
 * (Eq. 2) what falls outside its range.  Under that state L1BN + ReLU + Q_A
 * (Eq. 12-15) of an int8 code depends on (channel, code) only: the saved
 * per-(channel, code) A table.
 *
 * iseg_bn_infer -- A = table[c][z] for int8 codes z [M, C] whose exponent
 * must be the calibration's (ISEG_DEV_RANGE otherwise); *a_exp = the
 * calibration's A exponent.  C % 4 == 0, z and a_out 4-byte aligned.
 *
 * iseg_conv_bn_infer -- a conv layer with L1BN + ReLU? + Q_A in inference:
 * the conv's exact int32 sums (in the workspace), then one pass that puts
 * them on the calibration's Z grid (clamp(floor(sum 2^(e_x + e_w - e_Z) +
 * 1/2)) to 8 bits) and applies the A table.  saved: from iseg_bn_fwd on
 * that conv's output of a calibration batch; the geometry as for
 * iseg_conv_fwd; a_out [N, P, Q, K] int8. */
int iseg_bn_infer(const int8_t* z, const int32_t* z_exp, int64_t M, int64_t C, const void* saved,
                  int8_t* a_out, int32_t* a_exp, int32_t* dev_status, hipStream_t stream);
size_t iseg_conv_bn_infer_ws(const iseg_conv_geom* g);
int iseg_conv_bn_infer(const int8_t* x, const int32_t* x_exp, const int8_t* w, const int32_t* w_exp,
                       const iseg_conv_geom* g, const void* saved, int8_t* a_out, int32_t* a_exp,
                       void* ws, size_t ws_bytes, int32_t* dev_status, hipStream_t stream);

/* iseg_bn_fwd_i32 / iseg_bn_bwd_i32 -- the same L1BN forward and backward
 * (Eq. 12-15, 16) on the raw int32 sums of a convolution (iseg_conv_fwd with
 * ISEG_OUT_RAW), the literal dataflow of Sec. 3.2.2-3.2.3: BN takes the MAC
 * output before any activation quantizer, x-hat is quantized to k_xhat bits
 * because the bit width has grown, and Q_A (Eq. 15) follows BN.  Every
 * quantity is defined as for iseg_bn_fwd / iseg_bn_bwd; only the input is
 * wider.
 *   x [M, C] int32 with exponent s_x in [-40, 0] (ISEG_DEV_RANGE outside),
 *   M <= 2^22, C % 4 == 0.  saved: iseg_bn_i32_saved_bytes(C) bytes, its own
 *   layout (int32 hdr[16] = {b, y grid exponent, A exponent, s_x, A's shift},
 *   then each 256-byte aligned int32 n_mu[C], den[C], mlo[C], mhi[C]: the
 *   inputs with y > 0 form [mlo, mhi]).  The backward supports the exact E2
 *   (k_E2 >= 15) only (ISEG_ERR_UNSUPPORTED otherwise). */
size_t iseg_bn_i32_saved_bytes(int64_t C);
size_t iseg_bn_fwd_i32_ws(int64_t M, int64_t C);
int iseg_bn_fwd_i32(const int32_t* x, const int32_t* x_exp, int64_t M, int64_t C,
                    const int8_t* gamma_q, const int8_t* beta_q, const iseg_bn_cfg* cfg,
                    int8_t* y_out, int32_t* y_exp, void* saved,
                    void* ws, size_t ws_bytes, int32_t* dev_status, hipStream_t stream);
size_t iseg_bn_bwd_i32_ws(int64_t M, int64_t C);
int iseg_bn_bwd_i32(const int8_t* dy, const int32_t* dy_exp, const int32_t* x, int64_t M, int64_t C,
                    const int8_t* gamma_q, const iseg_bn_cfg* cfg, const void* saved, int8_t* dx_out,
                    int32_t* dx_exp, int64_t* dgamma, int64_t* dbeta, int32_t* dgamma_exp,
                    int32_t* dbeta_exp, void* ws, size_t ws_bytes, int32_t* dev_status,
                    hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Update (Eq. 19) and weight quantizer (Eq. 7-8)                            */
/* ------------------------------------------------------------------------ */

/* iseg_weight_update -- Delta W = UQ(G_q * 2^-lr_shift, k_U) (Eq. 19),
 * master <- clamp(master - Delta W, +-(2^(k_U-1)-1)), w_q = UQ(master, k_W)
 * (Eq. 8).  master [n] int32 codes with exponent master_exp (1-k_U for conv
 * weights; 2-k_U for gamma/beta, whose quantizers carry the x2 fold); g [n]
 * int8 codes with device exponent g_exp; w_q [n] int8 with exponent
 * master_exp + k_U - k_W.  k_U in [9, 31], k_W in [2, 8]. */
int iseg_weight_update(int32_t* master, int64_t n, const int8_t* g, const int32_t* g_exp,
                       int32_t lr_shift, int32_t master_exp, int32_t k_U, int32_t k_W,
                       int8_t* w_q, int32_t* dev_status, hipStream_t stream);

/* iseg_bn_param_update -- Q_G and Q_U of one L1BN layer's gamma and beta in
 * one launch: G = RQ(d, bits) keeping the scale (Eq. 5-6, 17) for d = dgamma
 * (Philox tensor id tid_gamma) and d = dbeta (tid_beta), Philox index = the
 * channel; then Delta = UQ(G 2^-lr_shift, k_U) (Eq. 19), master <- clamp(
 * master - Delta), and the quantized parameter UQ(master, k_W) (Eq. 14's
 * Q_gamma / Q_beta with the fixed x2 fold when master_exp = 2-k_U).  Equal to
 * iseg_requant (stochastic, keep_scale) followed by iseg_weight_update.
 *   dgamma, dbeta [C] int64 raw sums with device exponents; masters [C] int32
 *   (updated in place); gamma_q, beta_q [C] int8 out; g_gamma, g_beta [C] int8
 *   and g_*_exp (the quantized gradients) are optional outputs (NULL to skip). */
int iseg_bn_param_update(const int64_t* dgamma, const int32_t* dgamma_exp,
                         const int64_t* dbeta, const int32_t* dbeta_exp, int64_t C, int32_t bits,
                         uint64_t seed, uint32_t tid_gamma, uint32_t tid_beta, uint32_t step,
                         int32_t lr_shift, int32_t master_exp, int32_t k_U, int32_t k_W,
                         int32_t* gamma_m, int32_t* beta_m, int8_t* gamma_q, int8_t* beta_q,
                         int8_t* g_gamma, int8_t* g_beta, int32_t* g_gamma_exp, int32_t* g_beta_exp,
                         int32_t* dev_status, hipStream_t stream);

/* One parameter tensor of iseg_update_multi (a DEVICE array of these). */
enum iseg_update_kind {
    ISEG_UPD_CODES = 0,    /* g: int8 codes of a quantized gradient (conv weights after Q_G) */
    ISEG_UPD_RAW = 1       /* g: int64 raw sums (L1BN dgamma / dbeta); Q_G applied first */
};
typedef struct iseg_update_desc {
    int32_t* master;       /* k_U-bit master codes, updated in place */
    int8_t* w_q;           /* out: UQ(master, k_W) */
    const void* g;         /* gradient: int8 codes or int64 sums, see kind */
    const int32_t* g_exp;  /* device exponent of g */
    int8_t* g_q;           /* ISEG_UPD_RAW: out, the Q_G codes (may be NULL) */
    int32_t* g_q_exp;      /* ISEG_UPD_RAW: out, their exponent (may be NULL) */
    int64_t n;             /* elements; ISEG_UPD_RAW requires n <= 65536 */
    int32_t kind;          /* enum iseg_update_kind */
    int32_t master_exp;    /* 1-k_U for conv weights, 2-k_U for gamma / beta (x2 fold) */
    uint32_t tensor_id;    /* ISEG_UPD_RAW: Philox tensor id of Q_G */
    int32_t k_w;           /* code width of w_q for this tensor, 2..8 (k_W of conv
                              weights, k_gamma / k_beta of Sec. 3.2's BN); 0 = the
                              call's k_W.  Out of range: the entry is left as it
                              was and ISEG_DEV_DESC is set in *dev_status */
} iseg_update_desc;

/* iseg_update_multi -- the update step of a whole network in one launch: for
 * every descriptor, Q_G (ISEG_UPD_RAW: stochastic RQ to `bits` keeping the
 * scale, Eq. 5-6 and 17, Philox index = the element, key (seed, tensor_id),
 * counter step), then Delta = UQ(G 2^-lr_shift, k_U) (Eq. 19), master <-
 * clamp(master - Delta), w_q = UQ(master, k_W) (Eq. 8, or Eq. 14's fold for
 * gamma / beta; k_W per descriptor, see k_w).  Equal to iseg_weight_update
 * / iseg_bn_param_update per tensor.  descs: device array of n_desc <= 4096 descriptors (caller-owned;
 * the tensors they point to must not overlap). */
int iseg_update_multi(const iseg_update_desc* descs, int32_t n_desc, int32_t bits, uint64_t seed,
                      uint32_t step, int32_t lr_shift, int32_t k_U, int32_t k_W, int32_t* dev_status,
                      hipStream_t stream);

/* iseg_weight_quant -- Eq. 8 alone: w_q = UQ(master, k_W) from k_U-bit masters. */
int iseg_weight_quant(const int32_t* master, int64_t n, int32_t k_U, int32_t k_W,
                      int8_t* w_q, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Max pooling on codes (encoder glue)                                       */
/* ------------------------------------------------------------------------ */

/* iseg_maxpool_fwd -- window k x k, stride, zero-size padding never picked;
 * y [N,P,Q,C] with P = floor((H + 2 pad - k)/stride) + 1; y_exp = x_exp. */
int iseg_maxpool_fwd(const int8_t* x, const int32_t* x_exp, int64_t N, int64_t H, int64_t W,
                     int64_t C, int32_t k, int32_t stride, int32_t pad,
                     int8_t* y, int32_t* y_exp, hipStream_t stream);

/* iseg_maxpool_bwd -- each dy element goes to its window's first maximum in
 * row-major order; overlapping windows add exactly; then Q_E = SQ(., bits)
 * (Eq. 16).  dx [N,H,W,C] int8, dx_exp. */
size_t iseg_maxpool_bwd_ws(int64_t N, int64_t H, int64_t W, int64_t C);
int iseg_maxpool_bwd(const int8_t* dy, const int32_t* dy_exp, const int8_t* x,
                     int64_t N, int64_t H, int64_t W, int64_t C,
                     int32_t k, int32_t stride, int32_t pad, int32_t bits,
                     int8_t* dx, int32_t* dx_exp,
                     void* ws, size_t ws_bytes, int32_t* dev_status, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Merges of quantized tensors (residual add, error sums, ASPP concat, global */
/* pooling).  Every tensor of the dataflow is an 8-bit object with one scale */
/* (Sec. 3.1), so a merge forms the exact result on the grid 2^min(e_i) and   */
/* applies one SQ (Eq. 4; Eq. 16 for errors).  Exponents more than 48 apart   */
/* set ISEG_DEV_RANGE (outputs then unspecified).  Input arrays of pointers,  */
/* exponent pointers and per-input integers are HOST arrays of n_in entries   */
/* (n_in in [1, 8]) holding device pointers.                                  */
/* ------------------------------------------------------------------------ */

/* iseg_sum_requant -- out = SQ(ReLU?(sum_i in_i 2^(*in_exp[i] + exp_add[i])),
 * bits): the residual add of a bottleneck (relu = 1, the ReLU that follows
 * it) and the sum of the errors a tensor receives from several consumers
 * (relu = 0).  Input i is [N, HW, C] int8, or [N, 1, C] broadcast over the HW
 * positions when bcast[i] != 0 (the backward of global average pooling:
 * its error codes with exp_add = -log2(HW)).  exp_add and bcast may be NULL
 * (all zero).  out [N, HW, C] int8 with exponent *out_exp = min_i(e_i) + r,
 * r = bitlen(max|sum|) - (bits-1) (the minimum exponent itself for an
 * all-zero result).  bits in [2, 8]. */
size_t iseg_sum_requant_ws(int64_t N, int64_t HW, int64_t C);
int iseg_sum_requant(int32_t n_in, const int8_t* const* in, const int32_t* const* in_exp,
                     const int32_t* exp_add, const int32_t* bcast, int64_t N, int64_t HW, int64_t C,
                     int32_t relu, int32_t bits, int8_t* out, int32_t* out_exp,
                     void* ws, size_t ws_bytes, int32_t* dev_status, hipStream_t stream);

/* iseg_sum_requant_relu_mask -- the sum of the errors a residual add's output
 * receives (iseg_sum_requant with relu = 0, no broadcast inputs) followed by
 * the backward of that add's ReLU (iseg_relu_mask_bwd): out = the sum's codes
 * where sum_i mask_in_i 2^(*mask_exp[i]) > 0, else 0, with the sum's exponent
 * in *out_exp, bit-identical to the two calls in sequence, in two kernels
 * instead of three.  mask_in / mask_exp are host arrays of n_mask device
 * pointers (the add's inputs and their exponents), n_mask in [1, 8]; the
 * workspace is iseg_sum_requant_ws(N, HW, C).  Sec. 3.1, Eq. 16. */
int iseg_sum_requant_relu_mask(int32_t n_in, const int8_t* const* in, const int32_t* const* in_exp,
                               const int32_t* exp_add, int64_t N, int64_t HW, int64_t C, int32_t bits,
                               int32_t n_mask, const int8_t* const* mask_in, const int32_t* const* mask_exp,
                               int8_t* out, int32_t* out_exp, void* ws, size_t ws_bytes, int32_t* dev_status,
                               hipStream_t stream);

/* iseg_relu_mask_bwd -- backward of ReLU(sum_i in_i 2^(e_i + exp_add[i])):
 * dx = dy where the exact sum is > 0, else 0.  The values stay on dy's grid,
 * so dx takes dy's exponent (not written).  All tensors [n] int8, n a
 * multiple of the channel count C (C steers the vector path only). */
int iseg_relu_mask_bwd(const int8_t* dy, int32_t n_in, const int8_t* const* in,
                       const int32_t* const* in_exp, const int32_t* exp_add, int64_t n, int64_t C,
                       int8_t* dx, int32_t* dev_status, hipStream_t stream);

/* iseg_concat_requant -- out = SQ(concat_c(in_i 2^(*in_exp[i])), bits), one
 * object with one scale: the ASPP concatenation.  Input i is [N, HW, C_in[i]]
 * int8, or [N, 1, C_in[i]] broadcast over HW when bcast[i] != 0 (the image
 * pooling branch, whose 1x1 map is upsampled to the others' size); out
 * [N, HW, sum C_in] int8, *out_exp = min_i(e_i) + r. */
size_t iseg_concat_requant_ws(int32_t n_in);
int iseg_concat_requant(int32_t n_in, const int8_t* const* in, const int32_t* const* in_exp,
                        const int64_t* C_in, const int32_t* bcast, int64_t N, int64_t HW, int32_t bits,
                        int8_t* out, int32_t* out_exp, void* ws, size_t ws_bytes, int32_t* dev_status,
                        hipStream_t stream);

/* iseg_concat_split -- backward of the concatenation: out[i] [rows, C_in[i]]
 * = dy[:, off_i : off_i + C_in[i]] (off_i = sum of the earlier widths); the
 * slices keep dy's exponent.  A NULL out[i] is skipped (a broadcast part's
 * error is reduced by iseg_spatial_sum straight from dy instead). */
int iseg_concat_split(const int8_t* dy, int64_t rows, int32_t n_in, const int64_t* C_in,
                      int8_t* const* out, hipStream_t stream);

/* iseg_spatial_sum -- out[n, c] = SQ(sum_{hw} x[n, hw, c0 + c] / divisor, bits)
 * for x [N, HW, ldc] int8 with exponent *x_exp, c in [0, C): the scale is
 * 2^(x_exp + u), u the smallest integer with max|sum| < divisor 2^u, and
 * code = floor(sum 2^(bits-1-u) / divisor + 1/2) decided exactly.  Global
 * average pooling is divisor = HW (the exact mean); the backward of the mean
 * is HW = 1, divisor = the pooled H W (Q_E of dy / (H W), Eq. 16); the
 * backward of broadcasting a [N,1,C] tensor over HW positions is divisor = 1
 * (the exact spatial sum of the error, then Q_E).  out [N, C] int8; an
 * all-zero result has exponent *x_exp - ceil(log2 divisor).  Requires
 * N C <= 2^20, HW <= 2^23, divisor in [1, 2^30]. */
size_t iseg_spatial_sum_ws(int64_t N, int64_t HW, int64_t C);
int iseg_spatial_sum(const int8_t* x, const int32_t* x_exp, int64_t N, int64_t HW, int64_t ldc,
                     int64_t c0, int64_t C, int64_t divisor, int32_t bits, int8_t* out,
                     int32_t* out_exp, void* ws, size_t ws_bytes, int32_t* dev_status,
                     hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Segmentation loss (float region)                                          */
/* ------------------------------------------------------------------------ */

/* iseg_softmax_ce -- pixel-wise softmax cross-entropy of the logits
 * upsampled bilinearly to the label size (half-pixel centres: source
 * coordinate (o + 1/2) n_in / n_out - 1/2 clamped at 0, the upper neighbour
 * clamped at the edge), averaged over the N H W pixels; its gradient w.r.t.
 * the int8 logits (the adjoint of the upsampling applied to (softmax -
 * onehot) / (N H W)); and E1 = SQ(gradient, bits), the int8 error at the
 * logits (Eq. 4 / 16), exponent *err_exp.  Computed in float64.
 *   logits [N, h, w, K] int8 with exponent *logit_exp in [-1000, 0]
 *   (|logit| < 128: every exponential the region takes, of differences of
 *   at most 4 * 127 in magnitude, stays a normal finite double; outside it ISEG_DEV_RANGE, E1 codes 0, *loss NaN); a non-finite
 *   gradient sets ISEG_DEV_NONFINITE with the same outputs; labels [N, H, W]
 *   uint8 in [0, K) (otherwise ISEG_DEV_RANGE); loss: one device double
 *   (may be NULL); grad [N, h, w, K] device doubles (may be NULL); err
 *   [N, h, w, K] int8.  K <= 256, H >= h, W >= w. */
size_t iseg_softmax_ce_ws(int64_t N, int64_t h, int64_t w, int64_t K, int64_t H, int64_t W);
int iseg_softmax_ce(const int8_t* logits, const int32_t* logit_exp, const uint8_t* labels,
                    int64_t N, int64_t h, int64_t w, int64_t K, int64_t H, int64_t W, int32_t bits,
                    double* loss, double* grad, int8_t* err, int32_t* err_exp,
                    void* ws, size_t ws_bytes, int32_t* dev_status, hipStream_t stream);

/* iseg_mse_onehot -- the MSE loss of the network output against one-hot
 * labels (the FCN8s loss, Sec. 5.1): loss = mean over the N H W K elements of
 * (y - t)^2 with t = [k == label] (float64, summed per block and the block
 * partials in a fixed order), and E1 = SQ(2 (y - t) / (N H W K), bits) (Eq. 4
 * / 16) decided exactly (err codes, *err_exp).  y [N, H, W, K] int8 with
 * exponent *y_exp in [-60, 40] (ISEG_DEV_RANGE and a NaN loss outside);
 * labels [N, H, W] uint8 in [0, K) (otherwise ISEG_DEV_RANGE); loss: one
 * device double (may be NULL). */
size_t iseg_mse_onehot_ws(int64_t n);
int iseg_mse_onehot(const int8_t* y, const int32_t* y_exp, const uint8_t* labels, int64_t N, int64_t H,
                    int64_t W, int64_t K, int32_t bits, double* loss, int8_t* err, int32_t* err_exp,
                    void* ws, size_t ws_bytes, int32_t* dev_status, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Host-side utilities                                                       */
/* ------------------------------------------------------------------------ */

/* Philox4x32-10 block on the host, the same function the kernels use
 * (exposed for known-answer tests; no GPU needed). */
void iseg_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]);

/* Measurement hook.  Kernel families that can be timed in place: */
enum iseg_kernel_id {
    ISEG_KID_NONE = 0,
    ISEG_KID_CONV_FWD = 1,       /* every kernel of one iseg_conv_fwd call */
    ISEG_KID_CONV_BWD_DATA = 2,  /* every kernel of one iseg_conv_bwd_data call */
    ISEG_KID_CONV_WGRAD = 3,     /* every kernel of one iseg_conv_bwd_weight call */
    ISEG_KID_REQUANT = 4,        /* SQ/RQ code pass of any requantization */
    ISEG_KID_BN_FWD_APPLY = 5,   /* output pass of iseg_bn_fwd */
    ISEG_KID_BN_BWD_APPLY = 6,   /* output pass of iseg_bn_bwd */
    ISEG_KID_BN_FWD_STATS1 = 7,  /* first statistics pass of iseg_bn_fwd */
    ISEG_KID_BN_FWD_STATS2 = 8,  /* second statistics pass of iseg_bn_fwd */
    ISEG_KID_BN_BWD_STATS = 9,   /* statistics pass of iseg_bn_bwd */
    ISEG_KID_MAXPOOL_BWD = 10    /* routing pass of iseg_maxpool_bwd */
};

/* iseg_profile_arm -- the next launch of kernel family `kernel_id` (by any
 * entry point, on any stream; for the conv ids: the next call of that entry
 * point, all its kernels) records `start` immediately before and `stop`
 * immediately after itself on its own stream, then the hook disarms.  The
 * events are the caller's (hipEventCreate).  One arming per process: arming
 * again replaces it.  Thread-safe: exactly one launch claims an arming, even
 * when several threads launch at once.  kernel_id ISEG_KID_NONE disarms. */
int iseg_profile_arm(int32_t kernel_id, hipEvent_t start, hipEvent_t stop);

/* iseg_conv_last_plan -- the kernel path the calling thread's last
 * iseg_conv_fwd / iseg_conv_bwd_data(_t) / iseg_conv_bwd_weight call took:
 * "stem", "m32", "persist", "halo", "gemm_short", "conv_short",
 * "dma_two_pass", "dma_split", "dma_stage16", "dma" (raw sums), "igemm",
 * "wgrad_stem", "wgrad_taps", "wgrad_tr", "wgrad_atomic", or "none" when it
 * returned before choosing one.  Static storage, per thread.  For tests that
 * must reach a given kernel. */
const char* iseg_conv_last_plan(void);

/* ------------------------------------------------------------------------ */
/* Device status word                                                        */
/* ------------------------------------------------------------------------ */

/* iseg_status_read -- copy the sticky status word (device int32) to *value
 * (host) after the work already enqueued on `stream`; waits for the stream.
 * ISEG_ERR_DEVICE if the copy fails. */
int iseg_status_read(const int32_t* dev_status, int32_t* value, hipStream_t stream);

/* iseg_status_clear -- zero the status word on `stream` (a one-thread kernel,
 * so the call can sit in a captured graph). */
int iseg_status_clear(int32_t* dev_status, hipStream_t stream);

/* iseg_check_codes -- ISEG_DEV_RANGE in *dev_status if any of the n int8
 * codes of x (device, 16-byte aligned) lies outside [-(2^(bits-1)-1),
 * 2^(bits-1)-1] (Eq. 2's clip range), e.g. -128 in an 8-bit tensor from
 * outside the library. */
int iseg_check_codes(const int8_t* x, int64_t n, int32_t bits, int32_t* dev_status, hipStream_t stream);

/* Library version string (static storage). */
const char* iseg_version(void);

/* ------------------------------------------------------------------------ */
/* Step tape: native replay of a recorded sequence of calls                  */
/* ------------------------------------------------------------------------ */
/* A training step is a fixed sequence of the calls above on a few streams,
 * ordered by events, reading and writing the same buffers every step.  A
 * tape holds such a sequence, recorded once, and replays it from native code
 * (no per-call work of the caller's language runtime); it is how a caller
 * keeps the host side of a step short.  Nothing here is part of the paper's
 * method: it issues exactly the calls that were recorded.
 *
 * iseg_tape_entry -- index of an entry point by name (one of the int-returning
 *   compute calls above and iseg_profile_arm / iseg_status_clear /
 *   iseg_check_codes), or -1; iseg_tape_entry_nargs -- its parameter count.
 * iseg_tape_add_call -- append a call: words[n_words] are its arguments in
 *   declaration order, each as a 64-bit word (pointers and handles as
 *   addresses, integers sign- or zero-extended; the declared type is restored
 *   on replay).  blob (blob_bytes, a multiple of 8, host memory copied into the
 *   tape) holds the host structures and arrays the call reads through pointer
 *   arguments; the words listed in blob_words hold byte offsets into it and
 *   become addresses of the tape's copy.  step_word (-1: none) names the
 *   argument that carries the step counter of the stochastic rounding: on a
 *   run with step s it is step_base + s.  A recorded iseg_profile_arm becomes
 *   an armed slot (see iseg_tape_set_arm_events).
 * iseg_tape_add_record / iseg_tape_add_wait -- hipEventRecord(slot, stream) /
 *   hipStreamWaitEvent(stream, slot) on tape-owned events (created on first use).
 * iseg_tape_set_arm_events -- events[runs][n_arm][2] (start, stop) for the
 *   armed slots of the next `runs` runs, one set per run; an armed slot of any
 *   other run does nothing (the recorded events may no longer exist).
 * iseg_tape_run -- replay every operation in order on its recorded stream;
 *   stops at the first call that does not return ISEG_OK, returns that code
 *   and its index in *failed_op (-1 if none).  The caller keeps every buffer,
 *   stream and workspace the recorded calls use alive and unchanged in size,
 *   and must not run the same tape from two threads at once.
 * Memory: the tape itself lives in host memory (iseg_tape_create /
 *   iseg_tape_destroy, NULL if out of memory); its events are destroyed with it. */
void* iseg_tape_create(void);
void iseg_tape_destroy(void* tape);
int iseg_tape_entry(const char* name);
int iseg_tape_entry_nargs(int entry);
int iseg_tape_add_call(void* tape, int entry, const uint64_t* words, int n_words, const void* blob,
                       size_t blob_bytes, const int32_t* blob_words, int n_blob_words, int32_t step_word,
                       int64_t step_base);
int iseg_tape_add_record(void* tape, int32_t slot, hipStream_t stream);
int iseg_tape_add_wait(void* tape, hipStream_t stream, int32_t slot);
int iseg_tape_arm_count(const void* tape);
int iseg_tape_set_arm_events(void* tape, const hipEvent_t* events, int32_t runs);
int iseg_tape_run(void* tape, uint32_t step, int64_t* failed_op);
int64_t iseg_tape_size(const void* tape);

#ifdef __cplusplus
}
#endif

#endif /* ISEG_H */
