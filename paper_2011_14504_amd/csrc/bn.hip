// bn.hip -- L1 batch normalization (Eq. 12-15) and its backward on gfx950.
//
// Because the input of BN is an int8 code tensor, every per-element quantity
// of the forward (xhat_q, y, the ReLU mask, sgn(x - mu_q), the output code A)
// is a function of (channel, input code) only, and the backward's dx code is
// a function of (channel, sgn class, masked error code).  So the work splits
// into bandwidth-bound streaming passes over [M, C] (coalesced dword loads,
// four channels per lane, per-channel sums reduced through LDS and one global
// atomic per block and channel) and tiny finalize kernels that do the exact
// rational arithmetic (__int128) once per channel or per table entry.
//
// Forward:  stats1 (sum q, min q, max q) -> stats2 (sum |x - mu_q|) ->
//           fin1 (n_sigma, den, tensor max of |xhat|) -> fin2 (xhat codes,
//           y, max |y|) -> fin3 (A codes) -> apply (table gather).
// Backward: stats (sum delta, sum delta*xhat, sum sgn, per-class extremes of
//           delta) -> fin1 (dgamma, dbeta, max |gamma delta|) -> [stats2 for
//           k_E2 < 15] -> fin2 (max |dx|) -> table -> apply (gather).
#include "iseg_common.h"

namespace {

constexpr int kSentinelLo = -(1 << 30);

// ---------------------------------------------------------------------------
// saved-state layout (documented in iseg.h)
// ---------------------------------------------------------------------------
struct Saved {
    int32_t* hdr;
    int32_t *n_mu, *n_sigma, *den, *qmin, *qmax;
    int16_t* xcode;    // [C][256]
    uint8_t* flags;    // [C][256]
    int8_t* acode;     // [C][256]
};

size_t saved_bytes(int64_t C)
{
    return 256 + 5 * align256((size_t)C * 4) + align256((size_t)C * 512) +
           2 * align256((size_t)C * 256);
}

Saved saved_map(void* base, int64_t C)
{
    char* p = (char*)base;
    Saved s;
    s.hdr = (int32_t*)p; p += 256;
    s.n_mu = (int32_t*)p; p += align256((size_t)C * 4);
    s.n_sigma = (int32_t*)p; p += align256((size_t)C * 4);
    s.den = (int32_t*)p; p += align256((size_t)C * 4);
    s.qmin = (int32_t*)p; p += align256((size_t)C * 4);
    s.qmax = (int32_t*)p; p += align256((size_t)C * 4);
    s.xcode = (int16_t*)p; p += align256((size_t)C * 512);
    s.flags = (uint8_t*)p; p += align256((size_t)C * 256);
    s.acode = (int8_t*)p;
    return s;
}

// forward workspace
struct FwdWs {
    long long* S1;         // [C]
    long long* sumabs;     // [C]
    long long* Y;          // [C][256] y on the grid 2^e_y (before ReLU)
    int32_t* b_glob;       // tensor exponent of Q_xhat's scale (atomicMax)
    unsigned long long* maxY;
};

size_t fwd_ws_bytes(int64_t C)
{
    return 256 + 2 * align256((size_t)C * 8) + align256((size_t)C * 256 * 8);
}

FwdWs fwd_ws_map(void* base, int64_t C)
{
    char* p = (char*)base;
    FwdWs w;
    w.b_glob = (int32_t*)p;
    w.maxY = (unsigned long long*)(p + 64);
    p += 256;
    w.S1 = (long long*)p; p += align256((size_t)C * 8);
    w.sumabs = (long long*)p; p += align256((size_t)C * 8);
    w.Y = (long long*)p;
    return w;
}

// backward workspace
struct BwdWs {
    long long *sd, *sdn, *sf, *sfn;   // [C] sums of delta, delta*n_xhat, f, f*n_xhat
    int32_t* Z;                      // [C] sum of sgn(x - mu_q)
    int32_t* mm;                     // [C][6]: (min, max) delta for sgn = -1, 0, +1
    int8_t* lut;                     // [C][3][256] dx codes
    int32_t* bdx;                    // tensor exponent of E1's scale (atomicMax)
    unsigned long long* maxF;
};

size_t bwd_ws_bytes(int64_t C)
{
    return 256 + 4 * align256((size_t)C * 8) + align256((size_t)C * 4) +
           align256((size_t)C * 24) + align256((size_t)C * 768);
}

BwdWs bwd_ws_map(void* base, int64_t C)
{
    char* p = (char*)base;
    BwdWs w;
    w.bdx = (int32_t*)p;
    w.maxF = (unsigned long long*)(p + 64);
    p += 256;
    w.sd = (long long*)p; p += align256((size_t)C * 8);
    w.sdn = (long long*)p; p += align256((size_t)C * 8);
    w.sf = (long long*)p; p += align256((size_t)C * 8);
    w.sfn = (long long*)p; p += align256((size_t)C * 8);
    w.Z = (int32_t*)p; p += align256((size_t)C * 4);
    w.mm = (int32_t*)p; p += align256((size_t)C * 24);
    w.lut = (int8_t*)p;
    return w;
}

struct BnCfg {
    int32_t k_mu, k_sigma, k_xhat, k_gamma, k_beta, k_A, k_E1, k_E2, eps_code, relu;
};

BnCfg to_cfg(const iseg_bn_cfg* c)
{
    BnCfg b;
    b.k_mu = c->k_mu; b.k_sigma = c->k_sigma; b.k_xhat = c->k_xhat; b.k_gamma = c->k_gamma;
    b.k_beta = c->k_beta; b.k_A = c->k_A; b.k_E1 = c->k_E1; b.k_E2 = c->k_E2;
    b.eps_code = c->eps_code; b.relu = c->relu;
    return b;
}

// ---------------------------------------------------------------------------
// streaming geometry: a block covers one channel slice of CS channels (CS % 4
// == 0, CS divides C); lane g of a row handles channels 4g..4g+3 of the
// slice; rows_per_iter rows are in flight per block iteration.
// ---------------------------------------------------------------------------
struct Stream {
    int64_t M;
    int32_t C, CS, G, rpi;
};

__device__ __forceinline__ bool stream_lane(const Stream& st, int& g, int& rsub)
{
    g = threadIdx.x % st.G;
    rsub = threadIdx.x / st.G;
    return rsub < st.rpi;
}

int pick_cs(int64_t C, int csmax)
{
    for (int cs = csmax; cs >= 4; cs -= 4)
        if (C % cs == 0) return cs;
    return 0;
}

Stream make_stream(int64_t M, int64_t C, int cs)
{
    Stream s;
    s.M = M; s.C = (int32_t)C; s.CS = cs; s.G = cs / 4; s.rpi = 256 / s.G;
    return s;
}

dim3 stream_grid(const Stream& s)
{
    int nsl = s.C / s.CS;
    int64_t want = 2048 / nsl;
    if (want < 1) want = 1;
    int64_t rows = ceil_div64(s.M, s.rpi);
    int64_t gx = rows < want ? rows : want;
    if (gx < 1) gx = 1;
    return dim3((unsigned)gx, (unsigned)nsl);
}

__device__ __forceinline__ int sbyte(uint32_t w, int i) { return (int)(int8_t)(w >> (8 * i)); }

__device__ __forceinline__ bool sx_ok(int32_t s_x) { return s_x >= -40 && s_x <= 16; }

// D = (x - mu_q) / 2^g for code q; g = min(s_x, e_mu)
__device__ __forceinline__ int64_t bn_D(int q, int32_t s_x, int32_t n_mu, int e_mu)
{
    int g = s_x < e_mu ? s_x : e_mu;
    return (int64_t)q * ((int64_t)1 << (s_x - g)) - (int64_t)n_mu * ((int64_t)1 << (e_mu - g));
}

// n_mu from the channel sum (Eq. 14: mu_q = 2 UQ(mu/2, k_mu))
__device__ __forceinline__ int32_t bn_n_mu(long long S1, int32_t s_x, int64_t M, const BnCfg& cf)
{
    return (int32_t)clamp_k128(rhu128((i128)S1, s_x - 1 + (cf.k_mu - 1), (i128)M), cf.k_mu);
}

// ---------------------------------------------------------------------------
// forward kernels
// ---------------------------------------------------------------------------
__global__ void k_bnf_init(FwdWs w, Saved sv, int32_t C)
{
    int c = blockIdx.x * blockDim.x + threadIdx.x;
    if (c == 0) { *w.b_glob = kSentinelLo; *w.maxY = 0; }
    if (c < C) { w.S1[c] = 0; w.sumabs[c] = 0; sv.qmin[c] = 1000; sv.qmax[c] = -1000; }
}

__global__ __launch_bounds__(256) void k_bnf_stats1(const int8_t* __restrict__ x, Stream st, FwdWs w,
                                                    Saved sv)
{
    __shared__ int32_t sS[128], sMin[128], sMax[128];
    if (threadIdx.x < st.CS) { sS[threadIdx.x] = 0; sMin[threadIdx.x] = 1000; sMax[threadIdx.x] = -1000; }
    __syncthreads();
    int g, rsub;
    if (stream_lane(st, g, rsub)) {
        int s[4] = {0, 0, 0, 0}, mn[4] = {1000, 1000, 1000, 1000}, mx[4] = {-1000, -1000, -1000, -1000};
        int c0 = blockIdx.y * st.CS + g * 4;
        for (int64_t r = (int64_t)blockIdx.x * st.rpi + rsub; r < st.M; r += (int64_t)gridDim.x * st.rpi) {
            uint32_t v = *(const uint32_t*)(x + r * st.C + c0);
#pragma unroll
            for (int i = 0; i < 4; i++) {
                int q = sbyte(v, i);
                s[i] += q;
                mn[i] = q < mn[i] ? q : mn[i];
                mx[i] = q > mx[i] ? q : mx[i];
            }
        }
#pragma unroll
        for (int i = 0; i < 4; i++) {
            atomicAdd(&sS[g * 4 + i], s[i]);
            atomicMin(&sMin[g * 4 + i], mn[i]);
            atomicMax(&sMax[g * 4 + i], mx[i]);
        }
    }
    __syncthreads();
    if (threadIdx.x < st.CS) {
        int c = blockIdx.y * st.CS + threadIdx.x;
        atomicAdd((unsigned long long*)&w.S1[c], (unsigned long long)(long long)sS[threadIdx.x]);
        atomicMin(&sv.qmin[c], sMin[threadIdx.x]);
        atomicMax(&sv.qmax[c], sMax[threadIdx.x]);
    }
}

__global__ __launch_bounds__(256) void k_bnf_stats2(const int8_t* __restrict__ x, const int32_t* x_exp,
                                                    Stream st, FwdWs w, Saved sv, BnCfg cf,
                                                    int32_t* dev_status)
{
    __shared__ int32_t sMu[128];
    __shared__ unsigned long long sA[128];
    int32_t s_x = *x_exp;
    if (!sx_ok(s_x)) {
        if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) set_status(dev_status, ISEG_DEV_RANGE);
        return;
    }
    int e_mu = 2 - cf.k_mu;
    if (threadIdx.x < st.CS) {
        int c = blockIdx.y * st.CS + threadIdx.x;
        int32_t nm = bn_n_mu(w.S1[c], s_x, st.M, cf);
        sMu[threadIdx.x] = nm;
        sA[threadIdx.x] = 0;
        if (blockIdx.x == 0) sv.n_mu[c] = nm;
    }
    __syncthreads();
    int g, rsub;
    if (stream_lane(st, g, rsub)) {
        int c0 = blockIdx.y * st.CS + g * 4;
        int64_t a[4] = {0, 0, 0, 0};
        int gg = s_x < e_mu ? s_x : e_mu;
        int64_t mulq = (int64_t)1 << (s_x - gg);
        int64_t off[4];
#pragma unroll
        for (int i = 0; i < 4; i++) off[i] = (int64_t)sMu[g * 4 + i] * ((int64_t)1 << (e_mu - gg));
        for (int64_t r = (int64_t)blockIdx.x * st.rpi + rsub; r < st.M; r += (int64_t)gridDim.x * st.rpi) {
            uint32_t v = *(const uint32_t*)(x + r * st.C + c0);
#pragma unroll
            for (int i = 0; i < 4; i++) {
                int64_t D = (int64_t)sbyte(v, i) * mulq - off[i];
                a[i] += D < 0 ? -D : D;
            }
        }
#pragma unroll
        for (int i = 0; i < 4; i++) atomicAdd(&sA[g * 4 + i], (unsigned long long)a[i]);
    }
    __syncthreads();
    if (threadIdx.x < st.CS) {
        int c = blockIdx.y * st.CS + threadIdx.x;
        atomicAdd((unsigned long long*)&w.sumabs[c], sA[threadIdx.x]);
    }
}

// per channel: n_sigma, den, and this channel's bound on max|xhat|
__global__ void k_bnf_fin1(const int32_t* x_exp, int64_t M, int32_t C, FwdWs w, Saved sv, BnCfg cf)
{
    int c = blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= C) return;
    int32_t s_x = *x_exp;
    if (!sx_ok(s_x)) return;
    int e_mu = 2 - cf.k_mu, e_sig = 2 - cf.k_sigma;
    int gg = s_x < e_mu ? s_x : e_mu;
    // sigma/2 = sumabs 2^(g-1) / M ; n_sigma = floor(sigma/2 2^(k_sigma-1) + 1/2)
    int32_t ns = (int32_t)clamp_k128(rhu128((i128)w.sumabs[c], gg - 1 + (cf.k_sigma - 1), (i128)M), cf.k_sigma);
    int32_t den = ns + cf.eps_code;
    if (den < 1) den = 1;
    sv.n_sigma[c] = ns;
    sv.den[c] = den;
    int32_t nm = sv.n_mu[c];
    int best = kSentinelLo;
    int qs[2] = {sv.qmin[c], sv.qmax[c]};
    for (int t = 0; t < 2; t++) {
        int64_t D = bn_D(qs[t], s_x, nm, e_mu);
        if (D == 0) continue;
        int e = ceil_pow2_exp128(abs128((i128)D), (i128)den) + gg - e_sig;
        best = e > best ? e : best;
    }
    if (best > kSentinelLo) atomicMax(w.b_glob, best);
}

// per (channel, code): xhat code, y, flags; max |ReLU(y)| over the occurring codes
__global__ __launch_bounds__(256) void k_bnf_fin2(const int32_t* x_exp, FwdWs w, Saved sv, BnCfg cf,
                                                  const int8_t* gamma_q, const int8_t* beta_q)
{
    int c = blockIdx.x;
    int q = (int)threadIdx.x - 128;
    int32_t s_x = *x_exp;
    if (!sx_ok(s_x)) return;
    int b = *w.b_glob;
    if (b == kSentinelLo) b = 0;
    int e_mu = 2 - cf.k_mu, e_sig = 2 - cf.k_sigma;
    int e_g = 2 - cf.k_gamma, e_b = 2 - cf.k_beta;
    int e_xh = b - (cf.k_xhat - 1);
    int e_y = (e_g + e_xh) < e_b ? (e_g + e_xh) : e_b;
    int gg = s_x < e_mu ? s_x : e_mu;
    int64_t D = bn_D(q, s_x, sv.n_mu[c], e_mu);
    int32_t den = sv.den[c];
    i128 nx = clamp_k128(rhu128((i128)D, gg - e_sig + (cf.k_xhat - 1) - b, (i128)den), cf.k_xhat);
    i128 Y = (i128)gamma_q[c] * nx * pow2_128(e_g + e_xh - e_y) + (i128)beta_q[c] * pow2_128(e_b - e_y);
    int idx = c * 256 + threadIdx.x;
    sv.xcode[idx] = (int16_t)nx;
    int sg = (D > 0) - (D < 0);
    sv.flags[idx] = (uint8_t)((Y > 0 ? 1 : 0) | ((sg + 1) << 1));
    w.Y[idx] = (long long)Y;
    if (q == sv.qmin[c] || q == sv.qmax[c]) {
        i128 Yr = cf.relu && Y < 0 ? 0 : Y;
        atomicMax(w.maxY, (unsigned long long)abs128(Yr));
    }
}

__global__ __launch_bounds__(256) void k_bnf_fin3(const int32_t* x_exp, FwdWs w, Saved sv, BnCfg cf,
                                                  int32_t* y_exp)
{
    int c = blockIdx.x;
    int32_t s_x = *x_exp;
    if (!sx_ok(s_x)) return;
    int b = *w.b_glob;
    if (b == kSentinelLo) b = 0;
    int e_g = 2 - cf.k_gamma, e_b = 2 - cf.k_beta;
    int e_xh = b - (cf.k_xhat - 1);
    int e_y = (e_g + e_xh) < e_b ? (e_g + e_xh) : e_b;
    uint64_t M = *w.maxY;
    int r = M ? bitlen_u64(M) - (cf.k_A - 1) : 0;
    int idx = c * 256 + threadIdx.x;
    long long Y = w.Y[idx];
    if (cf.relu && Y < 0) Y = 0;
    sv.acode[idx] = (int8_t)sq_code(Y, r, cf.k_A);
    if (c == 0 && threadIdx.x == 0) {
        *y_exp = e_y + r;
        sv.hdr[0] = b;
        sv.hdr[1] = e_y;
        sv.hdr[2] = e_y + r;
        sv.hdr[3] = s_x;
    }
}

__global__ __launch_bounds__(256) void k_bnf_apply(const int8_t* __restrict__ x, int8_t* __restrict__ y,
                                                   Stream st, Saved sv)
{
    __shared__ int8_t lut[128 * 256];
    for (int i = threadIdx.x; i < st.CS * 64; i += blockDim.x)
        ((uint32_t*)lut)[i] = ((const uint32_t*)(sv.acode + (int64_t)blockIdx.y * st.CS * 256))[i];
    __syncthreads();
    int g, rsub;
    if (!stream_lane(st, g, rsub)) return;
    int c0 = blockIdx.y * st.CS + g * 4;
    const int8_t* l = lut + g * 4 * 256 + 128;
    for (int64_t r = (int64_t)blockIdx.x * st.rpi + rsub; r < st.M; r += (int64_t)gridDim.x * st.rpi) {
        uint32_t v = *(const uint32_t*)(x + r * st.C + c0);
        uint32_t o = 0;
#pragma unroll
        for (int i = 0; i < 4; i++) o |= (uint32_t)(uint8_t)l[i * 256 + sbyte(v, i)] << (8 * i);
        *(uint32_t*)(y + r * st.C + c0) = o;
    }
}

// ---------------------------------------------------------------------------
// backward kernels
// ---------------------------------------------------------------------------
__global__ void k_bnb_init(BwdWs w, int32_t C)
{
    int c = blockIdx.x * blockDim.x + threadIdx.x;
    if (c == 0) { *w.bdx = kSentinelLo; *w.maxF = 0; }
    if (c < C) {
        w.sd[c] = 0; w.sdn[c] = 0; w.sf[c] = 0; w.sfn[c] = 0; w.Z[c] = 0;
        for (int i = 0; i < 3; i++) { w.mm[c * 6 + 2 * i] = 1000; w.mm[c * 6 + 2 * i + 1] = -1000; }
    }
}

// pass 1: sum delta, sum delta*n_xhat, sum sgn, per-class min/max of delta
__global__ __launch_bounds__(256) void k_bnb_stats(const int8_t* __restrict__ dy,
                                                   const int8_t* __restrict__ x, Stream st, BwdWs w,
                                                   Saved sv, int32_t relu)
{
    __shared__ uint8_t fl[64 * 256];
    __shared__ int16_t xc[64 * 256];
    __shared__ unsigned long long sSd[64], sSdn[64];
    __shared__ int32_t sZ[64], sMM[64 * 6];
    int64_t cbase = (int64_t)blockIdx.y * st.CS;
    for (int i = threadIdx.x; i < st.CS * 256; i += blockDim.x) {
        fl[i] = sv.flags[cbase * 256 + i];
        xc[i] = sv.xcode[cbase * 256 + i];
    }
    if (threadIdx.x < st.CS) {
        sSd[threadIdx.x] = 0; sSdn[threadIdx.x] = 0; sZ[threadIdx.x] = 0;
        for (int i = 0; i < 3; i++) { sMM[threadIdx.x * 6 + 2 * i] = 1000; sMM[threadIdx.x * 6 + 2 * i + 1] = -1000; }
    }
    __syncthreads();
    int g, rsub;
    if (stream_lane(st, g, rsub)) {
        int c0 = (int)cbase + g * 4;
        int32_t sd[4] = {0, 0, 0, 0}, z[4] = {0, 0, 0, 0};
        int64_t sdn[4] = {0, 0, 0, 0};
        int32_t mm[4][6];
#pragma unroll
        for (int i = 0; i < 4; i++)
#pragma unroll
            for (int k = 0; k < 3; k++) { mm[i][2 * k] = 1000; mm[i][2 * k + 1] = -1000; }
        for (int64_t r = (int64_t)blockIdx.x * st.rpi + rsub; r < st.M; r += (int64_t)gridDim.x * st.rpi) {
            uint32_t vx = *(const uint32_t*)(x + r * st.C + c0);
            uint32_t vd = *(const uint32_t*)(dy + r * st.C + c0);
#pragma unroll
            for (int i = 0; i < 4; i++) {
                int li = (g * 4 + i) * 256 + sbyte(vx, i) + 128;
                int f = fl[li];
                int d = sbyte(vd, i);
                if (relu && !(f & 1)) d = 0;
                int cls = (f >> 1) & 3;           // sgn + 1
                sd[i] += d;
                sdn[i] += (int64_t)d * xc[li];
                z[i] += cls - 1;
#pragma unroll
                for (int k = 0; k < 3; k++)
                    if (cls == k) {
                        mm[i][2 * k] = d < mm[i][2 * k] ? d : mm[i][2 * k];
                        mm[i][2 * k + 1] = d > mm[i][2 * k + 1] ? d : mm[i][2 * k + 1];
                    }
            }
        }
#pragma unroll
        for (int i = 0; i < 4; i++) {
            int cl = g * 4 + i;
            atomicAdd(&sSd[cl], (unsigned long long)(long long)sd[i]);
            atomicAdd(&sSdn[cl], (unsigned long long)sdn[i]);
            atomicAdd(&sZ[cl], z[i]);
#pragma unroll
            for (int k = 0; k < 3; k++) {
                atomicMin(&sMM[cl * 6 + 2 * k], mm[i][2 * k]);
                atomicMax(&sMM[cl * 6 + 2 * k + 1], mm[i][2 * k + 1]);
            }
        }
    }
    __syncthreads();
    if (threadIdx.x < st.CS) {
        int c = (int)cbase + threadIdx.x;
        atomicAdd((unsigned long long*)&w.sd[c], sSd[threadIdx.x]);
        atomicAdd((unsigned long long*)&w.sdn[c], sSdn[threadIdx.x]);
        atomicAdd(&w.Z[c], sZ[threadIdx.x]);
        for (int k = 0; k < 3; k++) {
            atomicMin(&w.mm[c * 6 + 2 * k], sMM[threadIdx.x * 6 + 2 * k]);
            atomicMax(&w.mm[c * 6 + 2 * k + 1], sMM[threadIdx.x * 6 + 2 * k + 1]);
        }
    }
}

__global__ void k_bnb_fin1(const int32_t* dy_exp, int32_t C, BwdWs w, Saved sv, BnCfg cf,
                           const int8_t* gamma_q, int64_t* dgamma, int64_t* dbeta,
                           int32_t* dgamma_exp, int32_t* dbeta_exp, int32_t* dev_status)
{
    int c = blockIdx.x * blockDim.x + threadIdx.x;
    int32_t s_d = *dy_exp;
    if (c == 0) {
        if (s_d < -60 || s_d > 16) set_status(dev_status, ISEG_DEV_RANGE);
        *dbeta_exp = s_d;
        *dgamma_exp = s_d + sv.hdr[0] - (cf.k_xhat - 1);
    }
    if (c >= C) return;
    dbeta[c] = w.sd[c];
    dgamma[c] = w.sdn[c];
    int amax = 0;
    for (int k = 0; k < 3; k++) {
        int lo = w.mm[c * 6 + 2 * k], hi = w.mm[c * 6 + 2 * k + 1];
        if (lo > hi) continue;
        amax = (lo < 0 ? -lo : lo) > amax ? (lo < 0 ? -lo : lo) : amax;
        amax = (hi < 0 ? -hi : hi) > amax ? (hi < 0 ? -hi : hi) : amax;
    }
    int gq = gamma_q[c];
    uint64_t F = (uint64_t)(gq < 0 ? -gq : gq) * (uint64_t)amax;
    if (F) atomicMax(w.maxF, (unsigned long long)F);
}

__device__ __forceinline__ int bnb_r2(const BwdWs& w, const BnCfg& cf)
{
    uint64_t MF = *w.maxF;
    return MF ? bitlen_u64(MF) - (cf.k_E2 - 1) : 0;
}

// pass 2 (only when E2's quantizer rounds): sum f and f*n_xhat
__global__ __launch_bounds__(256) void k_bnb_stats2(const int8_t* __restrict__ dy,
                                                    const int8_t* __restrict__ x, Stream st, BwdWs w,
                                                    Saved sv, BnCfg cf, const int8_t* gamma_q)
{
    __shared__ uint8_t fl[64 * 256];
    __shared__ int16_t xc[64 * 256];
    __shared__ unsigned long long sF[64], sFn[64];
    int64_t cbase = (int64_t)blockIdx.y * st.CS;
    for (int i = threadIdx.x; i < st.CS * 256; i += blockDim.x) {
        fl[i] = sv.flags[cbase * 256 + i];
        xc[i] = sv.xcode[cbase * 256 + i];
    }
    if (threadIdx.x < st.CS) { sF[threadIdx.x] = 0; sFn[threadIdx.x] = 0; }
    __syncthreads();
    int r2 = bnb_r2(w, cf);
    int g, rsub;
    if (stream_lane(st, g, rsub)) {
        int c0 = (int)cbase + g * 4;
        int gq[4];
#pragma unroll
        for (int i = 0; i < 4; i++) gq[i] = gamma_q[c0 + i];
        int64_t sf[4] = {0, 0, 0, 0}, sfn[4] = {0, 0, 0, 0};
        for (int64_t r = (int64_t)blockIdx.x * st.rpi + rsub; r < st.M; r += (int64_t)gridDim.x * st.rpi) {
            uint32_t vx = *(const uint32_t*)(x + r * st.C + c0);
            uint32_t vd = *(const uint32_t*)(dy + r * st.C + c0);
#pragma unroll
            for (int i = 0; i < 4; i++) {
                int li = (g * 4 + i) * 256 + sbyte(vx, i) + 128;
                int d = sbyte(vd, i);
                if (cf.relu && !(fl[li] & 1)) d = 0;
                int64_t f = sq_code((int64_t)gq[i] * d, r2, cf.k_E2);
                sf[i] += f;
                sfn[i] += f * xc[li];
            }
        }
#pragma unroll
        for (int i = 0; i < 4; i++) {
            atomicAdd(&sF[g * 4 + i], (unsigned long long)sf[i]);
            atomicAdd(&sFn[g * 4 + i], (unsigned long long)sfn[i]);
        }
    }
    __syncthreads();
    if (threadIdx.x < st.CS) {
        int c = (int)cbase + threadIdx.x;
        atomicAdd((unsigned long long*)&w.sf[c], sF[threadIdx.x]);
        atomicAdd((unsigned long long*)&w.sfn[c], sFn[threadIdx.x]);
    }
}

// bracket of the exact dx (times den M^2 / 2^Ebase) for a (f, sgn) pair
__device__ __forceinline__ i128 bnb_bracket(int64_t f, int s, i128 M, i128 Sf, i128 T, i128 Z, int e_xh)
{
    i128 a = M * M * (i128)f - M * Sf;
    i128 t = T * (M * (i128)s - Z);
    return e_xh >= 0 ? a - (t << e_xh) : (a << -e_xh) - t;
}

struct BnbChan {
    i128 Sf, T, Z;
    int e_xh, Ebase, r2;
};

__device__ __forceinline__ BnbChan bnb_chan(int c, const int32_t* dy_exp, int64_t M, const BwdWs& w,
                                            const Saved& sv, const BnCfg& cf, int gq, bool exact_e2)
{
    BnbChan ch;
    ch.r2 = bnb_r2(w, cf);
    int b = sv.hdr[0];
    ch.e_xh = b - (cf.k_xhat - 1);
    int e_sig = 2 - cf.k_sigma, e_g = 2 - cf.k_gamma;
    int s2 = *dy_exp + e_g + ch.r2;
    ch.Ebase = s2 - e_sig + (ch.e_xh < 0 ? ch.e_xh : 0);
    if (exact_e2) {
        // E2 exact: f = gamma_q delta 2^-r2 with r2 <= 0
        ch.Sf = (i128)gq * (i128)w.sd[c] * pow2_128(-ch.r2);
        ch.T = (i128)gq * (i128)w.sdn[c] * pow2_128(-ch.r2);
    } else {
        ch.Sf = (i128)w.sf[c];
        ch.T = (i128)w.sfn[c];
    }
    ch.Z = (i128)w.Z[c];
    (void)M;
    return ch;
}

__global__ void k_bnb_fin2(const int32_t* dy_exp, int64_t M, int32_t C, BwdWs w, Saved sv, BnCfg cf,
                           const int8_t* gamma_q, int exact_e2)
{
    int c = blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= C) return;
    int gq = gamma_q[c];
    BnbChan ch = bnb_chan(c, dy_exp, M, w, sv, cf, gq, exact_e2);
    i128 Dd = (i128)sv.den[c] * (i128)M * (i128)M;
    int best = kSentinelLo;
    for (int k = 0; k < 3; k++) {
        int lo = w.mm[c * 6 + 2 * k], hi = w.mm[c * 6 + 2 * k + 1];
        if (lo > hi) continue;
        int ds[2] = {lo, hi};
        for (int t = 0; t < 2; t++) {
            int64_t f = sq_code((int64_t)gq * ds[t], ch.r2, cf.k_E2);
            i128 B = bnb_bracket(f, k - 1, (i128)M, ch.Sf, ch.T, ch.Z, ch.e_xh);
            if (B == 0) continue;
            int e = ceil_pow2_exp128(abs128(B), Dd) + ch.Ebase;
            best = e > best ? e : best;
        }
    }
    if (best > kSentinelLo) atomicMax(w.bdx, best);
}

// dx code table for every (sgn class, masked error code) of a channel
__global__ __launch_bounds__(256) void k_bnb_lut(const int32_t* dy_exp, int64_t M, BwdWs w, Saved sv,
                                                 BnCfg cf, const int8_t* gamma_q, int exact_e2,
                                                 int32_t* dx_exp)
{
    int c = blockIdx.x;
    int d = (int)threadIdx.x - 128;
    int gq = gamma_q[c];
    BnbChan ch = bnb_chan(c, dy_exp, M, w, sv, cf, gq, exact_e2);
    int bdx = *w.bdx;
    if (bdx == kSentinelLo) bdx = 0;
    if (c == 0 && threadIdx.x == 0) *dx_exp = bdx - (cf.k_E1 - 1);
    i128 Dd = (i128)sv.den[c] * (i128)M * (i128)M;
    int64_t f = d < -127 ? 0 : sq_code((int64_t)gq * d, ch.r2, cf.k_E2);
    for (int k = 0; k < 3; k++) {
        int8_t code = 0;
        if (d >= -127) {
            i128 B = bnb_bracket(f, k - 1, (i128)M, ch.Sf, ch.T, ch.Z, ch.e_xh);
            code = (int8_t)clamp_k128(rhu128(B, ch.Ebase + (cf.k_E1 - 1) - bdx, Dd), cf.k_E1);
        }
        w.lut[((int64_t)c * 3 + k) * 256 + threadIdx.x] = code;
    }
}

__global__ __launch_bounds__(256) void k_bnb_apply(const int8_t* __restrict__ dy,
                                                   const int8_t* __restrict__ x,
                                                   int8_t* __restrict__ dx, Stream st, BwdWs w,
                                                   Saved sv, int32_t relu)
{
    __shared__ uint8_t fl[64 * 256];
    __shared__ int8_t lut[64 * 768];
    int64_t cbase = (int64_t)blockIdx.y * st.CS;
    for (int i = threadIdx.x; i < st.CS * 64; i += blockDim.x)
        ((uint32_t*)fl)[i] = ((const uint32_t*)(sv.flags + cbase * 256))[i];
    for (int i = threadIdx.x; i < st.CS * 192; i += blockDim.x)
        ((uint32_t*)lut)[i] = ((const uint32_t*)(w.lut + cbase * 768))[i];
    __syncthreads();
    int g, rsub;
    if (!stream_lane(st, g, rsub)) return;
    int c0 = (int)cbase + g * 4;
    for (int64_t r = (int64_t)blockIdx.x * st.rpi + rsub; r < st.M; r += (int64_t)gridDim.x * st.rpi) {
        uint32_t vx = *(const uint32_t*)(x + r * st.C + c0);
        uint32_t vd = *(const uint32_t*)(dy + r * st.C + c0);
        uint32_t o = 0;
#pragma unroll
        for (int i = 0; i < 4; i++) {
            int cl = g * 4 + i;
            int f = fl[cl * 256 + sbyte(vx, i) + 128];
            int d = sbyte(vd, i);
            if (relu && !(f & 1)) d = 0;
            int cls = (f >> 1) & 3;
            o |= (uint32_t)(uint8_t)lut[(cl * 3 + cls) * 256 + d + 128] << (8 * i);
        }
        *(uint32_t*)(dx + r * st.C + c0) = o;
    }
}

bool cfg_ok(const iseg_bn_cfg* c)
{
    if (!c) return false;
    auto in = [](int v, int lo, int hi) { return v >= lo && v <= hi; };
    return in(c->k_mu, 2, 16) && in(c->k_sigma, 2, 16) && in(c->k_xhat, 2, 16) &&
           in(c->k_gamma, 2, 8) && in(c->k_beta, 2, 8) && in(c->k_A, 2, 8) && in(c->k_E1, 2, 8) &&
           in(c->k_E2, 2, 16) && in(c->eps_code, 0, 1 << 15) && (c->relu == 0 || c->relu == 1);
}

}  // namespace

// ---------------------------------------------------------------------------
// C ABI
// ---------------------------------------------------------------------------
extern "C" size_t iseg_bn_saved_bytes(int64_t C) { return C > 0 ? saved_bytes(C) : 0; }
extern "C" size_t iseg_bn_fwd_ws(int64_t, int64_t C) { return C > 0 ? fwd_ws_bytes(C) : 0; }
extern "C" size_t iseg_bn_bwd_ws(int64_t, int64_t C) { return C > 0 ? bwd_ws_bytes(C) : 0; }

extern "C" int iseg_bn_fwd(const int8_t* x, const int32_t* x_exp, int64_t M, int64_t C,
                           const int8_t* gamma_q, const int8_t* beta_q, const iseg_bn_cfg* cfg,
                           int8_t* y_out, int32_t* y_exp, void* saved,
                           void* ws, size_t ws_bytes, int32_t* dev_status, hipStream_t stream)
{
    if (M < 1 || C < 4) return ISEG_ERR_SHAPE;
    if (M > ((int64_t)1 << 22) || C > (1 << 16)) return ISEG_ERR_UNSUPPORTED;
    if (!x || !x_exp || !gamma_q || !beta_q || !y_out || !y_exp || !saved || !cfg_ok(cfg))
        return ISEG_ERR_ARG;
    int cs = pick_cs(C, 128);
    if (!cs || (((uintptr_t)x | (uintptr_t)y_out) & 3)) return ISEG_ERR_UNSUPPORTED;
    if (!ws || ws_bytes < fwd_ws_bytes(C)) return ISEG_ERR_WORKSPACE;
    BnCfg cf = to_cfg(cfg);
    Saved sv = saved_map(saved, C);
    FwdWs w = fwd_ws_map(ws, C);
    Stream st = make_stream(M, C, cs);
    dim3 sg = stream_grid(st);
    unsigned cg = (unsigned)ceil_div64(C, 256);
    hipLaunchKernelGGL(k_bnf_init, dim3(cg), dim3(256), 0, stream, w, sv, (int32_t)C);
    hipLaunchKernelGGL(k_bnf_stats1, sg, dim3(256), 0, stream, x, st, w, sv);
    hipLaunchKernelGGL(k_bnf_stats2, sg, dim3(256), 0, stream, x, x_exp, st, w, sv, cf, dev_status);
    hipLaunchKernelGGL(k_bnf_fin1, dim3(cg), dim3(256), 0, stream, x_exp, M, (int32_t)C, w, sv, cf);
    hipLaunchKernelGGL(k_bnf_fin2, dim3((unsigned)C), dim3(256), 0, stream, x_exp, w, sv, cf, gamma_q, beta_q);
    hipLaunchKernelGGL(k_bnf_fin3, dim3((unsigned)C), dim3(256), 0, stream, x_exp, w, sv, cf, y_exp);
    hipLaunchKernelGGL(k_bnf_apply, sg, dim3(256), 0, stream, x, y_out, st, sv);
    return launch_ok();
}

extern "C" int iseg_bn_bwd(const int8_t* dy, const int32_t* dy_exp, const int8_t* x,
                           int64_t M, int64_t C, const int8_t* gamma_q, const iseg_bn_cfg* cfg,
                           const void* saved, int8_t* dx_out, int32_t* dx_exp,
                           int64_t* dgamma, int64_t* dbeta, int32_t* dgamma_exp, int32_t* dbeta_exp,
                           void* ws, size_t ws_bytes, int32_t* dev_status, hipStream_t stream)
{
    if (M < 1 || C < 4) return ISEG_ERR_SHAPE;
    if (M > ((int64_t)1 << 22) || C > (1 << 16)) return ISEG_ERR_UNSUPPORTED;
    if (!dy || !dy_exp || !x || !gamma_q || !saved || !dx_out || !dx_exp || !dgamma || !dbeta ||
        !dgamma_exp || !dbeta_exp || !cfg_ok(cfg))
        return ISEG_ERR_ARG;
    int cs = pick_cs(C, 64);
    if (!cs || (((uintptr_t)x | (uintptr_t)dy | (uintptr_t)dx_out) & 3)) return ISEG_ERR_UNSUPPORTED;
    if (!ws || ws_bytes < bwd_ws_bytes(C)) return ISEG_ERR_WORKSPACE;
    BnCfg cf = to_cfg(cfg);
    Saved sv = saved_map((void*)saved, C);
    BwdWs w = bwd_ws_map(ws, C);
    Stream st = make_stream(M, C, cs);
    dim3 sg = stream_grid(st);
    unsigned cg = (unsigned)ceil_div64(C, 256);
    // E2 = SQ(gamma delta, k_E2) is exact when |gamma delta| <= 127^2 < 2^(k_E2-1)
    int exact_e2 = cf.k_E2 >= 15;
    hipLaunchKernelGGL(k_bnb_init, dim3(cg), dim3(256), 0, stream, w, (int32_t)C);
    hipLaunchKernelGGL(k_bnb_stats, sg, dim3(256), 0, stream, dy, x, st, w, sv, cf.relu);
    hipLaunchKernelGGL(k_bnb_fin1, dim3(cg), dim3(256), 0, stream, dy_exp, (int32_t)C, w, sv, cf,
                       gamma_q, dgamma, dbeta, dgamma_exp, dbeta_exp, dev_status);
    if (!exact_e2)
        hipLaunchKernelGGL(k_bnb_stats2, sg, dim3(256), 0, stream, dy, x, st, w, sv, cf, gamma_q);
    hipLaunchKernelGGL(k_bnb_fin2, dim3(cg), dim3(256), 0, stream, dy_exp, M, (int32_t)C, w, sv, cf,
                       gamma_q, exact_e2);
    hipLaunchKernelGGL(k_bnb_lut, dim3((unsigned)C), dim3(256), 0, stream, dy_exp, M, w, sv, cf,
                       gamma_q, exact_e2, dx_exp);
    hipLaunchKernelGGL(k_bnb_apply, sg, dim3(256), 0, stream, dy, x, dx_out, st, w, sv, cf.relu);
    return launch_ok();
}
