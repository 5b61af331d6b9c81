/*
 * iseg_oracle.c -- plain CPU oracle for the integer training dataflow of
 * "Training and Inference for Integer-Based Semantic Segmentation Network"
 * (arXiv 2011.14504).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, obviously-correct
 * reference that the GPU library is checked against.  Only the tests, the
 * smoke check and the benchmark's CPU-baseline leg may load it.  It shares no
 * code, header or table with the GPU library.
 *
 * Representation used throughout: a quantized object is a tensor of integer
 * codes n together with ONE power-of-two exponent e per tensor, so that the
 * real value is n * 2^e (Sec. 3.1: a scale per quantized object).
 *
 * Arithmetic is exact: int64 and __int128, plain loops, no blocking and no
 * lookup tables.  Every function names the equation it follows.  Readings of
 * the paper where it is silent or ambiguous are listed in the design notes and
 * repeated at the function that applies them.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>

typedef __int128 i128;
typedef unsigned __int128 u128;

enum {
    ORC_OK = 0,
    ORC_ERR_ARG = 1,
    ORC_ERR_RANGE = 6,
};

/* ------------------------------------------------------------------------ */
/* exact integer helpers                                                     */
/* ------------------------------------------------------------------------ */

static i128 i128_abs(i128 v) { return v < 0 ? -v : v; }

/* number of significant bits of |v| (0 for v == 0) */
static int bitlen(i128 v)
{
    u128 a = (u128)i128_abs(v);
    int b = 0;
    while (a) { b++; a >>= 1; }
    return b;
}

/* mathematical floor(a / b) for b > 0 */
static i128 floor_div(i128 a, i128 b)
{
    i128 q = a / b;
    if ((a % b) != 0 && a < 0) q -= 1;
    return q;
}

static i128 p2(int e) { return (i128)1 << e; }

/* floor(num * 2^sh / den + 1/2) for den > 0: "round half up", the rounding of
 * Eq. 2 (floor of x/Delta + 1/2). */
static i128 round_half_up(i128 num, int sh, i128 den)
{
    if (sh >= 0)
        return floor_div(2 * num * p2(sh) + den, 2 * den);
    return floor_div(2 * num + den * p2(-sh), 2 * den * p2(-sh));
}

/* |A| < B * 2^t  for A >= 0, B > 0 */
static int lt_scaled(i128 A, i128 B, int t)
{
    if (t >= 0) return A < B * p2(t);
    return A * p2(-t) < B;
}

/* smallest integer e with A < B * 2^e  (A >= 0, B > 0): the exponent of the
 * smallest power of two strictly greater than A/B. */
static int ceil_pow2_exp(i128 A, i128 B)
{
    int e = bitlen(A) - bitlen(B);
    while (!lt_scaled(A, B, e)) e++;
    while (lt_scaled(A, B, e - 1)) e--;
    return e;
}

static i128 clamp_code(i128 v, int k)
{
    i128 lim = p2(k - 1) - 1;          /* UQ clips to [-1+Delta, 1-Delta] */
    if (v > lim) return lim;
    if (v < -lim) return -lim;
    return v;
}

/* ------------------------------------------------------------------------ */
/* Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11), written from its        */
/* published definition: 10 rounds of the 4x32 S-box with multipliers        */
/* 0xD2511F53 / 0xCD9E8D57 and Weyl key increments 0x9E3779B9 / 0xBB67AE85.  */
/* ------------------------------------------------------------------------ */
void orc_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4])
{
    uint32_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
    uint32_t k0 = key_in[0], k1 = key_in[1];
    for (int round = 0; round < 10; round++) {
        uint64_t p0 = (uint64_t)0xD2511F53u * c0;
        uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        uint32_t n0 = hi1 ^ c1 ^ k0;
        uint32_t n1 = lo1;
        uint32_t n2 = hi0 ^ c3 ^ k1;
        uint32_t n3 = lo0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* The uniform draw used by stochastic rounding for element `idx` of tensor
 * `tensor_id`: key = (seed mod 2^32, tensor_id), counter = (idx mod 2^32,
 * idx >> 32, step, 0); the 64-bit draw is w0 | w1 << 32. */
uint64_t orc_draw_u64(uint64_t seed, uint32_t tensor_id, uint32_t step, uint64_t idx)
{
    uint32_t ctr[4] = { (uint32_t)idx, (uint32_t)(idx >> 32), step, 0u };
    uint32_t key[2] = { (uint32_t)seed, tensor_id };
    uint32_t o[4];
    orc_philox4x32_10(ctr, key, o);
    return (uint64_t)o[0] | ((uint64_t)o[1] << 32);
}

/* ------------------------------------------------------------------------ */
/* Eq. 1-2: uniform quantizer on a real number held exactly in a double.     */
/* Delta(k) = 2^(1-k); UQ(x,k) = Clip(Delta*floor(x/Delta + 1/2), -1+Delta,   */
/* 1-Delta).  Returned as the integer code n with UQ = n * Delta.            */
/* ------------------------------------------------------------------------ */
int64_t orc_uq_code_f64(double x, int k)
{
    double v = ldexp(x, k - 1);        /* x / Delta, exact (power-of-two scale) */
    double fl = floor(v);
    double frac = v - fl;              /* exact for |v| < 2^52 */
    double n = fl + (frac >= 0.5 ? 1.0 : 0.0);
    double lim = ldexp(1.0, k - 1) - 1.0;
    if (n > lim) n = lim;
    if (n < -lim) n = -lim;
    return (int64_t)n;
}

/* iseg_quantize oracle on float32 input.
 * mode 0 = UQ (Eq. 2): code = UQ(x, k) / Delta, exponent 1-k.
 * mode 1 = SQ (Eq. 4) with the power-of-two reading of Scale (Eq. 3):
 *          S = 2^b, the smallest power of two strictly greater than max|x|;
 *          code = UQ(x/S, k)/Delta, exponent b+1-k.  All-zero input -> codes 0,
 *          exponent 1-k.
 * Non-finite inputs are rejected. */
int orc_quantize_f32(const float* x, int64_t n, int k, int mode,
                     int64_t* codes, int32_t* exp_out)
{
    if (k < 2 || k > 31 || n < 0) return ORC_ERR_ARG;
    double M = 0.0;
    for (int64_t i = 0; i < n; i++) {
        if (!isfinite(x[i])) return ORC_ERR_RANGE;
        double a = fabs((double)x[i]);
        if (a > M) M = a;
    }
    int b = 0;
    if (mode == 1) {
        if (M > 0.0) {
            int e;
            frexp(M, &e);          /* M = f * 2^e, f in [0.5, 1): 2^e is the
                                      smallest power of two strictly above M */
            b = e;
        }
    } else if (mode != 0) {
        return ORC_ERR_ARG;
    }
    for (int64_t i = 0; i < n; i++)
        codes[i] = orc_uq_code_f64(ldexp((double)x[i], -b), k);
    *exp_out = b + 1 - k;
    return ORC_OK;
}

/* The same quantizer on float64 input (the loss gradient of the float
 * softmax region is held in double precision): identical rules, the decision
 * floor(v + 1/2) taken exactly on the double value. */
int orc_quantize_f64(const double* x, int64_t n, int k, int mode,
                     int64_t* codes, int32_t* exp_out)
{
    if (k < 2 || k > 31 || n < 0) return ORC_ERR_ARG;
    double M = 0.0;
    for (int64_t i = 0; i < n; i++) {
        if (!isfinite(x[i])) return ORC_ERR_RANGE;
        double a = fabs(x[i]);
        if (a > M) M = a;
    }
    int b = 0;
    if (mode == 1) {
        if (M > 0.0) {
            int e;
            frexp(M, &e);
            b = e;
        }
    } else if (mode != 0) {
        return ORC_ERR_ARG;
    }
    for (int64_t i = 0; i < n; i++)
        codes[i] = orc_uq_code_f64(ldexp(x[i], -b), k);
    *exp_out = b + 1 - k;
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Eq. 4 (SQ) and Eq. 5-6 (RQ) on an integer tensor with exponent in_exp.    */
/* Scale(x) (Eq. 3) read as the smallest power of two strictly greater than  */
/* max|x|: S = 2^(bitlen(M) + in_exp).  With r = bitlen(M) - (k-1):           */
/*   SQ code = clamp(floor(q / 2^r + 1/2))                                    */
/*   RQ code = clamp(floor(q / 2^r) + [U < q/2^r - floor(q/2^r)])             */
/* U is the top r bits of the Philox draw of the element (uniform in         */
/* {0..2^r-1}/2^r), so P(round up) is exactly the fractional part (Eq. 6).   */
/* For r <= 0 the division is exact: the code is q * 2^-r for both modes.     */
/* Exponent: keep_scale=1 -> in_exp + r (Eq. 4, Eq. 17); keep_scale=0 ->      */
/* 1-k, the scale dropped (Eq. 18).  All-zero input: codes 0, exponent in_exp */
/* (keep) or 1-k (drop).                                                      */
/* ------------------------------------------------------------------------ */
int orc_requant(const int64_t* in, int64_t n, int32_t in_exp, int k,
                int stochastic, int keep_scale,
                uint64_t seed, uint32_t tensor_id, uint32_t step,
                int64_t* codes, int32_t* exp_out)
{
    if (k < 2 || k > 31 || n < 0) return ORC_ERR_ARG;
    i128 M = 0;
    for (int64_t i = 0; i < n; i++) {
        i128 a = i128_abs((i128)in[i]);
        if (a > M) M = a;
    }
    if (M == 0) {
        for (int64_t i = 0; i < n; i++) codes[i] = 0;
        *exp_out = keep_scale ? in_exp : 1 - k;
        return ORC_OK;
    }
    int r = bitlen(M) - (k - 1);
    for (int64_t i = 0; i < n; i++) {
        i128 q = in[i];
        i128 c;
        if (r <= 0) {
            c = q * p2(-r);
        } else if (!stochastic) {
            c = round_half_up(q, -r, 1);
        } else {
            i128 fl = floor_div(q, p2(r));
            i128 rem = q - fl * p2(r);           /* numerator of the fraction */
            uint64_t u = orc_draw_u64(seed, tensor_id, step, (uint64_t)i);
            i128 ur = (i128)(u >> (64 - r));     /* top r bits */
            c = fl + (ur < rem ? 1 : 0);
        }
        codes[i] = (int64_t)clamp_code(c, k);
    }
    *exp_out = keep_scale ? in_exp + r : 1 - k;
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Convolutions: exact integer sums, zero padding, cross-correlation, NHWC    */
/* activations and KRSC weights.  Output size                                */
/*   P = floor((H + 2 pad - dil (R-1) - 1) / stride) + 1.                      */
/* geom = {N,H,W,C,K,R,S, stride_h,stride_w, pad_h,pad_w, dil_h,dil_w}        */
/* ------------------------------------------------------------------------ */
static int64_t out_dim(int64_t H, int64_t R, int64_t st, int64_t pad, int64_t dil)
{
    return (H + 2 * pad - dil * (R - 1) - 1) / st + 1;
}

/* forward: acc[n,p,q,k] = sum_{r,s,c} x[n, p*st-pad+r*d, q*st-pad+s*d, c] * w[k,r,s,c] */
void orc_conv_fwd_raw(const int8_t* x, const int8_t* w, const int64_t* g, int64_t* acc)
{
    int64_t N = g[0], H = g[1], W = g[2], C = g[3], K = g[4], R = g[5], S = g[6];
    int64_t sh = g[7], sw = g[8], ph = g[9], pw = g[10], dh = g[11], dw = g[12];
    int64_t P = out_dim(H, R, sh, ph, dh), Q = out_dim(W, S, sw, pw, dw);
    #pragma omp parallel for collapse(2) schedule(static)
    for (int64_t n = 0; n < N; n++)
    for (int64_t p = 0; p < P; p++)
    for (int64_t q = 0; q < Q; q++)
    for (int64_t k = 0; k < K; k++) {
        int64_t sum = 0;
        for (int64_t r = 0; r < R; r++) {
            int64_t h = p * sh - ph + r * dh;
            if (h < 0 || h >= H) continue;
            for (int64_t s = 0; s < S; s++) {
                int64_t ww = q * sw - pw + s * dw;
                if (ww < 0 || ww >= W) continue;
                const int8_t* xp = x + ((n * H + h) * W + ww) * C;
                const int8_t* wp = w + ((k * R + r) * S + s) * C;
                for (int64_t c = 0; c < C; c++) sum += (int64_t)xp[c] * (int64_t)wp[c];
            }
        }
        acc[((n * P + p) * Q + q) * K + k] = sum;
    }
}

/* backward-data, the adjoint of the forward map (Eq. 16 takes its SQ):
 *   dx[n,h,w,c] = sum over (p,q,k,r,s) with h = p*st-pad+r*d, w = q*st-pad+s*d
 *                 of dy[n,p,q,k] * w[k,r,s,c]
 * written as the literal scatter of every forward product term. */
void orc_conv_bwd_data_raw(const int8_t* dy, const int8_t* w, const int64_t* g, int64_t* dx)
{
    int64_t N = g[0], H = g[1], W = g[2], C = g[3], K = g[4], R = g[5], S = g[6];
    int64_t sh = g[7], sw = g[8], ph = g[9], pw = g[10], dh = g[11], dw = g[12];
    int64_t P = out_dim(H, R, sh, ph, dh), Q = out_dim(W, S, sw, pw, dw);
    memset(dx, 0, sizeof(int64_t) * (size_t)(N * H * W * C));
    #pragma omp parallel for schedule(static)
    for (int64_t n = 0; n < N; n++)
    for (int64_t p = 0; p < P; p++)
    for (int64_t q = 0; q < Q; q++)
    for (int64_t k = 0; k < K; k++) {
        int64_t e = dy[((n * P + p) * Q + q) * K + k];
        if (e == 0) continue;
        for (int64_t r = 0; r < R; r++) {
            int64_t h = p * sh - ph + r * dh;
            if (h < 0 || h >= H) continue;
            for (int64_t s = 0; s < S; s++) {
                int64_t ww = q * sw - pw + s * dw;
                if (ww < 0 || ww >= W) continue;
                int64_t* xp = dx + ((n * H + h) * W + ww) * C;
                const int8_t* wp = w + ((k * R + r) * S + s) * C;
                for (int64_t c = 0; c < C; c++) xp[c] += e * (int64_t)wp[c];
            }
        }
    }
}

/* backward-weight (the gradient G of Eq. 17-18 before quantization):
 *   dw[k,r,s,c] = sum_{n,p,q} dy[n,p,q,k] * x[n, p*st-pad+r*d, q*st-pad+s*d, c] */
void orc_conv_bwd_weight_raw(const int8_t* dy, const int8_t* x, const int64_t* g, int64_t* dw_out)
{
    int64_t N = g[0], H = g[1], W = g[2], C = g[3], K = g[4], R = g[5], S = g[6];
    int64_t sh = g[7], sw = g[8], ph = g[9], pw = g[10], dh = g[11], dw = g[12];
    int64_t P = out_dim(H, R, sh, ph, dh), Q = out_dim(W, S, sw, pw, dw);
    #pragma omp parallel for collapse(2) schedule(static)
    for (int64_t k = 0; k < K; k++)
    for (int64_t r = 0; r < R; r++)
    for (int64_t s = 0; s < S; s++) {
        int64_t* out = dw_out + ((k * R + r) * S + s) * C;
        for (int64_t c = 0; c < C; c++) out[c] = 0;
        for (int64_t n = 0; n < N; n++)
        for (int64_t p = 0; p < P; p++) {
            int64_t h = p * sh - ph + r * dh;
            if (h < 0 || h >= H) continue;
            for (int64_t q = 0; q < Q; q++) {
                int64_t ww = q * sw - pw + s * dw;
                if (ww < 0 || ww >= W) continue;
                int64_t e = dy[((n * P + p) * Q + q) * K + k];
                if (e == 0) continue;
                const int8_t* xp = x + ((n * H + h) * W + ww) * C;
                for (int64_t c = 0; c < C; c++) out[c] += e * (int64_t)xp[c];
            }
        }
    }
}

/* ------------------------------------------------------------------------ */
/* L1 batch normalization, forward (Eq. 12-15).                               */
/*                                                                            */
/* Input: integer codes q (NHWC flattened to M rows x C channels), exponent */
/* s_x: int8 codes of a requantized conv output, or the conv's raw int32    */
/* sums (the wide input of the literal dataflow, orc_bn_fwd32).            */
/* Per channel c over its m = M values:                                       */
/*   mu     = (1/m) sum x                                     (Eq. 10)        */
/*   mu_q   = 2 UQ(mu/2, k_mu)        -> code n_mu, value n_mu 2^(2-k_mu)     */
/*   sigma  = (1/m) sum |x - mu_q|                            (Eq. 13)        */
/*   sigma_q= 2 UQ(sigma/2, k_sigma)  -> code n_sigma, value n_sigma 2^(2-k_s)*/
/*   xhat   = (x - mu_q) / (sigma_q + eps)                    (Eq. 12)        */
/*   xhat_q = SQ(xhat, k_xhat), one scale for the whole tensor                */
/*   y      = gamma_q xhat_q + beta_q  (gamma_q = n_g 2^(2-k_g), same for beta)*/
/*   y      = ReLU(y) if relu                                                  */
/*   A      = SQ(y, k_A)                                      (Eq. 15)        */
/* Readings: sigma uses the quantized mean mu_q; eps = eps_code LSBs of the   */
/* sigma grid and the denominator code is max(n_sigma + eps_code, 1); ReLU    */
/* sits between the affine step and Q_A; SQ uses the power-of-two scale; an   */
/* all-zero xhat takes b = 0 (exponent 1-k_xhat).                             */
/* Preconditions (else ORC_ERR_RANGE): s_x in [-40, 16], 1 <= m <= 2^22.      */
/* Why 16: with g = min(s_x, e_mu) = -14 for s_x >= -14, a centred value     */
/* D = q 2^(s_x+14) - n_mu has |D| <= 127 2^30 + 32767 < 2^37 at s_x = 16,    */
/* so the per-channel sum of |D| over m <= 2^22 rows stays below 2^59: a     */
/* signed 64-bit accumulator (the GPU keeps these partial sums in int64)     */
/* with four bits to spare.  At s_x = 20 the same sum could reach           */
/* 127 2^34 2^22 ~ 2^63 and overflow.  Every other intermediate is smaller:  */
/* |xhat| < 2^37 (b <= 37), y on its grid < 2^44, and the backward bracket   */
/* m^2 f - m sum f - (sum f n_xhat) 2^(b-15) (m s - Z) < 2^96 in __int128.   */
/* s_x = -40 keeps 2^(e_mu - g) = 2^26 and the sum of |D| likewise in range. */
/* Raw int32 input (|q| < 2^31): s_x in [-40, 0], so |D| < 2^46, the sum of  */
/* |D| < 2^68 (held in __int128 here), |xhat| < 2^46 (b <= 46), y < 2^54 on  */
/* its grid and the backward bracket < 2^106.                               */
/* ------------------------------------------------------------------------ */
typedef struct {
    int k_mu, k_sigma, k_xhat, k_gamma, k_beta, k_A, k_E1, k_E2, eps_code, relu;
} orc_bn_cfg;

/* per-channel forward statistics shared by the forward and backward oracles */
typedef struct {
    int64_t n_mu, n_sigma, den;
    int g;               /* exponent of the grid on which D = x - mu_q is an integer */
} orc_bn_chan;

static int bn_channel_stats(const int32_t* x, int32_t s_x, int64_t M, int64_t C, int64_t c,
                            const orc_bn_cfg* cf, orc_bn_chan* st)
{
    int e_mu = 2 - cf->k_mu, e_sig = 2 - cf->k_sigma;
    i128 S1 = 0;
    for (int64_t i = 0; i < M; i++) S1 += x[i * C + c];
    /* mu/2 = S1 2^(s_x - 1) / m ; code = floor(mu/2 * 2^(k_mu-1) + 1/2) */
    i128 n_mu = clamp_code(round_half_up(S1, s_x - 1 + (cf->k_mu - 1), M), cf->k_mu);
    int g = s_x < e_mu ? s_x : e_mu;
    i128 sumabs = 0;
    for (int64_t i = 0; i < M; i++) {
        i128 D = (i128)x[i * C + c] * p2(s_x - g) - n_mu * p2(e_mu - g);
        sumabs += i128_abs(D);
    }
    /* sigma/2 = sumabs 2^(g-1) / m */
    i128 n_sigma = clamp_code(round_half_up(sumabs, g - 1 + (cf->k_sigma - 1), M), cf->k_sigma);
    i128 den = n_sigma + cf->eps_code;
    if (den < 1) den = 1;
    st->n_mu = (int64_t)n_mu;
    st->n_sigma = (int64_t)n_sigma;
    st->den = (int64_t)den;
    st->g = g;
    (void)e_sig;
    return ORC_OK;
}

/* D_i = (x_i - mu_q) / 2^g, an exact integer */
static i128 bn_D(int32_t q, int32_t s_x, const orc_bn_chan* st, int e_mu)
{
    return (i128)q * p2(s_x - st->g) - (i128)st->n_mu * p2(e_mu - st->g);
}

/* xhat_i = D_i 2^(g - e_sigma) / den : returns numerator D, the power of two,
 * and den via the channel stats.  The tensor exponent b of Q_xhat:
 * smallest b with max|xhat| < 2^b. */
static int bn_fwd_core(const int32_t* x, int32_t s_x, int wide, int64_t M, int64_t C,
                       const int8_t* gq, const int8_t* bq, const orc_bn_cfg* cf,
                       orc_bn_chan* st, int* b_out, int16_t* nxh /* M*C */,
                       i128* Y /* M*C, pre-ReLU y on grid 2^e_y */, int* e_y_out)
{
    if (s_x < -40 || s_x > (wide ? 0 : 16) || M < 1 || M > ((int64_t)1 << 22)) return ORC_ERR_RANGE;
    int e_mu = 2 - cf->k_mu, e_sig = 2 - cf->k_sigma;
    for (int64_t c = 0; c < C; c++) bn_channel_stats(x, s_x, M, C, c, cf, &st[c]);
    /* b = smallest integer with |xhat_i| < 2^b for all i */
    int have = 0, b = 0;
    for (int64_t c = 0; c < C; c++) {
        for (int64_t i = 0; i < M; i++) {
            i128 D = bn_D(x[i * C + c], s_x, &st[c], e_mu);
            if (D == 0) continue;
            /* |D| 2^(g - e_sig) / den < 2^e  <=>  |D| < den 2^(e - g + e_sig) */
            int t = ceil_pow2_exp(i128_abs(D), st[c].den);
            int e = t + st[c].g - e_sig;
            if (!have || e > b) { b = e; have = 1; }
        }
    }
    /* Q_xhat = SQ(xhat, k_xhat): n = clamp(floor(xhat 2^(k-1-b) + 1/2)) */
    int kx = cf->k_xhat;
    int e_xh = b - (kx - 1);                       /* exponent of xhat_q */
    int e_g = 2 - cf->k_gamma, e_b = 2 - cf->k_beta;
    int e_y = (e_g + e_xh) < e_b ? (e_g + e_xh) : e_b;
    for (int64_t c = 0; c < C; c++) {
        for (int64_t i = 0; i < M; i++) {
            i128 D = bn_D(x[i * C + c], s_x, &st[c], e_mu);
            i128 n = clamp_code(round_half_up(D, st[c].g - e_sig + (kx - 1) - b, st[c].den), kx);
            nxh[i * C + c] = (int16_t)n;
            /* y = gamma_q xhat_q + beta_q on the grid 2^e_y */
            Y[i * C + c] = (i128)gq[c] * n * p2(e_g + e_xh - e_y) + (i128)bq[c] * p2(e_b - e_y);
        }
    }
    *b_out = b;
    *e_y_out = e_y;
    return ORC_OK;
}

static int bn_fwd_any(const int32_t* x, int32_t s_x, int wide, int64_t M, int64_t C,
                      const int8_t* gq, const int8_t* bq, const int32_t* cfg_arr,
                      int8_t* out, int32_t* out_exp,
                      int32_t* n_mu, int32_t* n_sigma, int32_t* b_xhat, int16_t* nxh_out)
{
    orc_bn_cfg cf = { cfg_arr[0], cfg_arr[1], cfg_arr[2], cfg_arr[3], cfg_arr[4],
                      cfg_arr[5], cfg_arr[6], cfg_arr[7], cfg_arr[8], cfg_arr[9] };
    orc_bn_chan* st = (orc_bn_chan*)calloc((size_t)C, sizeof(orc_bn_chan));
    int16_t* nxh = (int16_t*)malloc(sizeof(int16_t) * (size_t)(M * C));
    i128* Y = (i128*)malloc(sizeof(i128) * (size_t)(M * C));
    int b = 0, e_y = 0;
    int rc = bn_fwd_core(x, s_x, wide, M, C, gq, bq, &cf, st, &b, nxh, Y, &e_y);
    if (rc == ORC_OK) {
        /* ReLU, then A = SQ(y, k_A) with one power-of-two scale per tensor */
        i128 Mx = 0;
        for (int64_t i = 0; i < M * C; i++) {
            if (cf.relu && Y[i] < 0) Y[i] = 0;
            if (i128_abs(Y[i]) > Mx) Mx = i128_abs(Y[i]);
        }
        int r = Mx == 0 ? 0 : bitlen(Mx) - (cf.k_A - 1);
        for (int64_t i = 0; i < M * C; i++) {
            i128 v = r > 0 ? round_half_up(Y[i], -r, 1) : Y[i] * p2(-r);
            out[i] = (int8_t)clamp_code(v, cf.k_A);
        }
        *out_exp = e_y + r;
        for (int64_t c = 0; c < C; c++) {
            if (n_mu) n_mu[c] = (int32_t)st[c].n_mu;
            if (n_sigma) n_sigma[c] = (int32_t)st[c].n_sigma;
        }
        if (b_xhat) *b_xhat = b;
        if (nxh_out) memcpy(nxh_out, nxh, sizeof(int16_t) * (size_t)(M * C));
    }
    free(st); free(nxh); free(Y);
    return rc;
}

/* int8 codes widened to int32 (exact), for the one core of both inputs */
static int32_t* widen8(const int8_t* x, int64_t n)
{
    int32_t* w = (int32_t*)malloc(sizeof(int32_t) * (size_t)(n > 0 ? n : 1));
    for (int64_t i = 0; i < n; i++) w[i] = x[i];
    return w;
}

int orc_bn_fwd(const int8_t* x, int32_t s_x, int64_t M, int64_t C,
               const int8_t* gq, const int8_t* bq, const int32_t* cfg_arr,
               int8_t* out, int32_t* out_exp,
               int32_t* n_mu, int32_t* n_sigma, int32_t* b_xhat, int16_t* nxh_out)
{
    int32_t* w = widen8(x, M * C);
    int rc = bn_fwd_any(w, s_x, 0, M, C, gq, bq, cfg_arr, out, out_exp, n_mu, n_sigma, b_xhat, nxh_out);
    free(w);
    return rc;
}

/* the same forward on the raw int32 sums of a convolution */
int orc_bn_fwd32(const int32_t* x, int32_t s_x, int64_t M, int64_t C,
                 const int8_t* gq, const int8_t* bq, const int32_t* cfg_arr,
                 int8_t* out, int32_t* out_exp,
                 int32_t* n_mu, int32_t* n_sigma, int32_t* b_xhat, int16_t* nxh_out)
{
    return bn_fwd_any(x, s_x, 1, M, C, gq, bq, cfg_arr, out, out_exp, n_mu, n_sigma, b_xhat, nxh_out);
}

/* ------------------------------------------------------------------------ */
/* L1 batch normalization, backward.  The paper prints no formula; this is    */
/* the exact derivative of Eq. 12-13 with straight-through estimators across */
/* Q_mu, Q_sigma, Q_xhat and Q_A, and sgn(0) = 0:                             */
/*   delta  = dA * [y > 0]            (ReLU mask from y before Q_A)           */
/*   dbeta  = sum delta,  dgamma = sum delta * xhat_q        (raw, per chan)  */
/*   E2     = SQ(gamma_q * delta, k_E2)            (Eq. 16, error at xhat)    */
/*   dx_i   = [E2_i - mean(E2) - mean(E2 xhat_q) (s_i - mean(s))]             */
/*            / (sigma_q + eps),      s_i = sgn(x_i - mu_q)                   */
/*   E1     = SQ(dx, k_E1)                         (Eq. 16, error at input)   */
/* Means run over the channel's m values; SQ scales are per tensor.           */
/* Derivation: d mu/dx_j = 1/m, d sigma/dx_j = (s_j - mean(s))/m, so          */
/*   d xhat_i/dx_j = [(delta_ij - 1/m) - xhat_i (s_j - mean(s))/m]/(sigma+eps)*/
/* Optional dx_pre receives the value of dx before E1's quantizer (double).   */
/* ------------------------------------------------------------------------ */
static int bn_bwd_any(const int8_t* dA, int32_t s_d, const int32_t* x, int32_t s_x, int wide,
                      int64_t M, int64_t C, const int8_t* gq, const int8_t* bq,
                      const int32_t* cfg_arr,
                      int8_t* dx, int32_t* dx_exp,
                      int64_t* dgamma, int64_t* dbeta, int32_t* dgamma_exp, int32_t* dbeta_exp,
                      double* dx_pre, int64_t* zero_sum_failures)
{
    orc_bn_cfg cf = { cfg_arr[0], cfg_arr[1], cfg_arr[2], cfg_arr[3], cfg_arr[4],
                      cfg_arr[5], cfg_arr[6], cfg_arr[7], cfg_arr[8], cfg_arr[9] };
    if (s_d < -60 || s_d > 20) return ORC_ERR_RANGE;
    orc_bn_chan* st = (orc_bn_chan*)calloc((size_t)C, sizeof(orc_bn_chan));
    int16_t* nxh = (int16_t*)malloc(sizeof(int16_t) * (size_t)(M * C));
    i128* Y = (i128*)malloc(sizeof(i128) * (size_t)(M * C));
    i128* F = (i128*)malloc(sizeof(i128) * (size_t)(M * C));
    i128* B = (i128*)malloc(sizeof(i128) * (size_t)(M * C));
    int b = 0, e_y = 0;
    int rc = bn_fwd_core(x, s_x, wide, M, C, gq, bq, &cf, st, &b, nxh, Y, &e_y);
    if (rc != ORC_OK) goto done;
    {
        int e_mu = 2 - cf.k_mu, e_sig = 2 - cf.k_sigma, e_g = 2 - cf.k_gamma;
        int e_xh = b - (cf.k_xhat - 1);
        /* delta with the ReLU mask; parameter gradients */
        for (int64_t c = 0; c < C; c++) {
            i128 sb = 0, sg = 0;
            for (int64_t i = 0; i < M; i++) {
                int64_t j = i * C + c;
                i128 d = dA[j];
                if (cf.relu && !(Y[j] > 0)) d = 0;
                F[j] = d;                       /* delta for now */
                sb += d;
                sg += d * nxh[j];
            }
            dbeta[c] = (int64_t)sb;
            dgamma[c] = (int64_t)sg;
        }
        *dbeta_exp = s_d;
        *dgamma_exp = s_d + e_xh;
        /* E2 = SQ(gamma_q * delta, k_E2): integers F on grid 2^(s_d + e_g) */
        i128 MF = 0;
        for (int64_t c = 0; c < C; c++)
            for (int64_t i = 0; i < M; i++) {
                int64_t j = i * C + c;
                F[j] = (i128)gq[c] * F[j];
                if (i128_abs(F[j]) > MF) MF = i128_abs(F[j]);
            }
        int r2 = MF == 0 ? 0 : bitlen(MF) - (cf.k_E2 - 1);
        int s2 = s_d + e_g + r2;
        for (int64_t j = 0; j < M * C; j++) {
            i128 v = r2 > 0 ? round_half_up(F[j], -r2, 1) : F[j] * p2(-r2);
            F[j] = clamp_code(v, cf.k_E2);   /* f_j : E2_j = f_j 2^s2 */
        }
        /* dx_i = 2^(s2 - e_sig) / (den m^2) * [m^2 f_i - m Sf - T 2^e_xh (m s_i - Z)]
         * with Sf = sum f, T = sum f n_xhat, Z = sum s.  For e_xh < 0 the bracket
         * is multiplied through by 2^-e_xh. */
        int have = 0, bdx = 0;
        int64_t zfail = 0;
        int Ebase = s2 - e_sig + (e_xh < 0 ? e_xh : 0);
        for (int64_t c = 0; c < C; c++) {
            i128 m = M, Sf = 0, T = 0, Z = 0;
            for (int64_t i = 0; i < M; i++) {
                int64_t j = i * C + c;
                i128 D = bn_D(x[j], s_x, &st[c], e_mu);
                Sf += F[j];
                T += F[j] * nxh[j];
                Z += (D > 0) - (D < 0);
            }
            i128 bsum = 0;
            for (int64_t i = 0; i < M; i++) {
                int64_t j = i * C + c;
                i128 D = bn_D(x[j], s_x, &st[c], e_mu);
                i128 s = (D > 0) - (D < 0);
                i128 a = m * m * F[j] - m * Sf;
                i128 t = T * (m * s - Z);
                i128 Bn = e_xh >= 0 ? a - t * p2(e_xh) : a * p2(-e_xh) - t;
                B[j] = Bn;
                bsum += Bn;
                if (Bn != 0) {
                    /* |dx| = |Bn| 2^Ebase / (den m^2) < 2^e */
                    int e = ceil_pow2_exp(i128_abs(Bn), (i128)st[c].den * m * m) + Ebase;
                    if (!have || e > bdx) { bdx = e; have = 1; }
                }
                if (dx_pre)
                    dx_pre[j] = ldexp((double)Bn / ((double)st[c].den * (double)M * (double)M), Ebase);
            }
            if (bsum != 0) zfail++;
        }
        if (zero_sum_failures) *zero_sum_failures = zfail;
        /* E1 = SQ(dx, k_E1) */
        int k1 = cf.k_E1;
        for (int64_t c = 0; c < C; c++) {
            i128 Dd = (i128)st[c].den * (i128)M * (i128)M;
            for (int64_t i = 0; i < M; i++) {
                int64_t j = i * C + c;
                i128 v = round_half_up(B[j], Ebase + (k1 - 1) - bdx, Dd);
                dx[j] = (int8_t)clamp_code(v, k1);
            }
        }
        *dx_exp = bdx - (k1 - 1);
    }
done:
    free(st); free(nxh); free(Y); free(F); free(B);
    return rc;
}

int orc_bn_bwd(const int8_t* dA, int32_t s_d, const int8_t* x, int32_t s_x,
               int64_t M, int64_t C, const int8_t* gq, const int8_t* bq,
               const int32_t* cfg_arr,
               int8_t* dx, int32_t* dx_exp,
               int64_t* dgamma, int64_t* dbeta, int32_t* dgamma_exp, int32_t* dbeta_exp,
               double* dx_pre, int64_t* zero_sum_failures)
{
    int32_t* w = widen8(x, M * C);
    int rc = bn_bwd_any(dA, s_d, w, s_x, 0, M, C, gq, bq, cfg_arr, dx, dx_exp, dgamma, dbeta, dgamma_exp,
                        dbeta_exp, dx_pre, zero_sum_failures);
    free(w);
    return rc;
}

/* the backward of orc_bn_fwd32 (raw int32 conv sums as the input) */
int orc_bn_bwd32(const int8_t* dA, int32_t s_d, const int32_t* x, int32_t s_x,
                 int64_t M, int64_t C, const int8_t* gq, const int8_t* bq,
                 const int32_t* cfg_arr,
                 int8_t* dx, int32_t* dx_exp,
                 int64_t* dgamma, int64_t* dbeta, int32_t* dgamma_exp, int32_t* dbeta_exp,
                 double* dx_pre, int64_t* zero_sum_failures)
{
    return bn_bwd_any(dA, s_d, x, s_x, 1, M, C, gq, bq, cfg_arr, dx, dx_exp, dgamma, dbeta, dgamma_exp,
                      dbeta_exp, dx_pre, zero_sum_failures);
}

/* ------------------------------------------------------------------------ */
/* Inference with frozen statistics (the paper claims fixed-point inference  */
/* but gives no rule for running statistics).  Reading: a layer's inference  */
/* state is captured from one calibration forward in training mode -- per   */
/* channel n_mu and n_sigma, and the exponents of the conv output Z, of     */
/* Q_xhat's scale (b) and of Q_A -- and every later input uses that state:  */
/* no batch statistic and no data-dependent scale, so each quantizer is a   */
/* fixed-step UQ that clips what falls outside its range.                   */
/* ------------------------------------------------------------------------ */

/* codes = clamp(floor(a 2^(a_exp - out_exp) + 1/2), k bits): a quantizer with
 * a fixed step 2^out_exp (half-up rounding, Eq. 2's clip) */
int orc_requant_fixed(const int64_t* in, int64_t n, int32_t in_exp, int32_t out_exp, int k, int64_t* codes)
{
    if (k < 2 || k > 31 || n < 0 || in_exp - out_exp > 60 || out_exp - in_exp > 100) return ORC_ERR_ARG;
    int sh = in_exp - out_exp;
    for (int64_t i = 0; i < n; i++)
        codes[i] = (int64_t)clamp_code(round_half_up((i128)in[i], sh, 1), k);
    return ORC_OK;
}

/* L1BN + ReLU? + Q_A of int8 codes z (exponent s_x) with the frozen state:
 * mu_q = n_mu 2^(2-k_mu), sigma_q = n_sigma 2^(2-k_sigma) per channel, x-hat
 * on the fixed grid 2^(b+1-k_xhat), A on the fixed grid 2^a_exp:
 *   xhat_q = UQ-like clamp(floor((x - mu_q)/(sigma_q + eps) 2^(k_xhat-1-b) + 1/2))
 *   y      = gamma_q xhat_q + beta_q, ReLU if cfg->relu
 *   A      = clamp(floor(y 2^-a_exp + 1/2), k_A bits)                        */
int orc_bn_infer(const int8_t* x, int32_t s_x, int64_t M, int64_t C,
                 const int8_t* gq, const int8_t* bq, const int32_t* cfg_arr,
                 const int32_t* n_mu, const int32_t* n_sigma, int32_t b, int32_t a_exp, int8_t* out)
{
    orc_bn_cfg cf = { cfg_arr[0], cfg_arr[1], cfg_arr[2], cfg_arr[3], cfg_arr[4],
                      cfg_arr[5], cfg_arr[6], cfg_arr[7], cfg_arr[8], cfg_arr[9] };
    if (s_x < -40 || s_x > 16 || M < 0) return ORC_ERR_RANGE;
    int e_mu = 2 - cf.k_mu, e_sig = 2 - cf.k_sigma;
    int e_xh = b - (cf.k_xhat - 1);
    int e_g = 2 - cf.k_gamma, e_b = 2 - cf.k_beta;
    int e_y = (e_g + e_xh) < e_b ? (e_g + e_xh) : e_b;
    for (int64_t c = 0; c < C; c++) {
        orc_bn_chan st;
        st.n_mu = n_mu[c];
        st.n_sigma = n_sigma[c];
        st.den = n_sigma[c] + cf.eps_code;
        if (st.den < 1) st.den = 1;
        st.g = s_x < e_mu ? s_x : e_mu;
        for (int64_t i = 0; i < M; i++) {
            int64_t j = i * C + c;
            i128 D = bn_D(x[j], s_x, &st, e_mu);
            i128 n = clamp_code(round_half_up(D, st.g - e_sig + (cf.k_xhat - 1) - b, st.den), cf.k_xhat);
            i128 Y = (i128)gq[c] * n * p2(e_g + e_xh - e_y) + (i128)bq[c] * p2(e_b - e_y);
            if (cf.relu && Y < 0) Y = 0;
            out[j] = (int8_t)clamp_code(round_half_up(Y, e_y - a_exp, 1), cf.k_A);
        }
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Eq. 19 (Q_U) and Eq. 8 (Q_W): master update and re-quantized weights.     */
/*   Delta W = UQ(G_q * lr, k_U)  with lr = 2^-lr_shift                       */
/*   W_m    <- clamp(W_m - Delta W)          (master held at k_U bits)        */
/*   W_q    = UQ(W_m, k_W)                                                     */
/* master codes have exponent master_exp: 1-k_U for conv weights; 2-k_U for   */
/* gamma/beta, whose quantizers carry the fixed x2 fold (Q_gamma = 2 UQ(./2)).*/
/* w_q exponent = master_exp + (k_U - k_W).                                   */
/* ------------------------------------------------------------------------ */
int orc_weight_update(int32_t* master, int64_t n, const int8_t* gcode, int32_t g_exp,
                      int lr_shift, int master_exp, int k_U, int k_W, int8_t* w_q)
{
    if (k_U < 2 || k_U > 31 || k_W < 2 || k_W > 8 || k_W > k_U) return ORC_ERR_ARG;
    int sh = g_exp - lr_shift - master_exp;
    for (int64_t i = 0; i < n; i++) {
        i128 g = gcode[i];
        i128 dW;
        if (g == 0) dW = 0;
        else if (sh > 40) dW = g > 0 ? p2(k_U - 1) - 1 : -(p2(k_U - 1) - 1);
        else dW = clamp_code(round_half_up(g, sh, 1), k_U);
        i128 m = clamp_code((i128)master[i] - dW, k_U);
        master[i] = (int32_t)m;
        w_q[i] = (int8_t)clamp_code(round_half_up(m, -(k_U - k_W), 1), k_W);
    }
    return ORC_OK;
}

/* Eq. 8 alone: W_q = UQ(W_m, k_W) */
int orc_weight_quant(const int32_t* master, int64_t n, int k_U, int k_W, int8_t* w_q)
{
    if (k_U < 2 || k_U > 31 || k_W < 2 || k_W > 8 || k_W > k_U) return ORC_ERR_ARG;
    for (int64_t i = 0; i < n; i++)
        w_q[i] = (int8_t)clamp_code(round_half_up((i128)master[i], -(k_U - k_W), 1), k_W);
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Max pooling on codes (glue of the VGG16 / ResNet50 encoders).  Forward     */
/* picks the first maximum in row-major window order; padding is never      */
/* picked.  Backward routes each output error to that position; overlapping  */
/* windows add up exactly (the caller then applies SQ, Eq. 16).              */
/* ------------------------------------------------------------------------ */
static int64_t pool_argmax(const int8_t* x, int64_t H, int64_t W, int64_t C,
                           int64_t n, int64_t p, int64_t q, int64_t c,
                           int64_t k, int64_t st, int64_t pad)
{
    int64_t best = -1;
    int bv = -1000;
    for (int64_t r = 0; r < k; r++) {
        int64_t h = p * st - pad + r;
        if (h < 0 || h >= H) continue;
        for (int64_t s = 0; s < k; s++) {
            int64_t w = q * st - pad + s;
            if (w < 0 || w >= W) continue;
            int64_t idx = ((n * H + h) * W + w) * C + c;
            if (x[idx] > bv) { bv = x[idx]; best = idx; }
        }
    }
    return best;
}

void orc_maxpool_fwd(const int8_t* x, int64_t N, int64_t H, int64_t W, int64_t C,
                     int64_t k, int64_t st, int64_t pad, int8_t* y)
{
    int64_t P = (H + 2 * pad - k) / st + 1, Q = (W + 2 * pad - k) / st + 1;
    for (int64_t n = 0; n < N; n++)
    for (int64_t p = 0; p < P; p++)
    for (int64_t q = 0; q < Q; q++)
    for (int64_t c = 0; c < C; c++)
        y[((n * P + p) * Q + q) * C + c] = x[pool_argmax(x, H, W, C, n, p, q, c, k, st, pad)];
}

void orc_maxpool_bwd_raw(const int8_t* dy, const int8_t* x, int64_t N, int64_t H, int64_t W,
                         int64_t C, int64_t k, int64_t st, int64_t pad, int64_t* dx)
{
    int64_t P = (H + 2 * pad - k) / st + 1, Q = (W + 2 * pad - k) / st + 1;
    memset(dx, 0, sizeof(int64_t) * (size_t)(N * H * W * C));
    for (int64_t n = 0; n < N; n++)
    for (int64_t p = 0; p < P; p++)
    for (int64_t q = 0; q < Q; q++)
    for (int64_t c = 0; c < C; c++)
        dx[pool_argmax(x, H, W, C, n, p, q, c, k, st, pad)] += dy[((n * P + p) * Q + q) * C + c];
}

int orc_num_threads(void)
{
#ifdef _OPENMP
    extern int omp_get_max_threads(void);
    return omp_get_max_threads();
#else
    return 1;
#endif
}
