// conv.hip -- int8 x int8 -> int32 convolutions on gfx950 MFMA.
//
// All three passes are implicit GEMMs over NHWC activations / KRSC weights:
//   forward     rows = output pixels (n,p,q), cols = K, reduction = (r,s,c)
//   bwd-data    rows = input pixels  (n,h,w), cols = C, reduction = (r,s,k)
//   bwd-weight  rows = K, cols = (r,s,c), reduction = output pixels (n,p,q)
// The forward and backward-data passes share one kernel: the reduction runs
// tap-major with the channel index innermost, so a 16-byte piece of the A
// tile is a contiguous channel run of one gathered pixel (zero when the tap
// falls into padding, or for bwd-data when the stride does not divide it).
// Tiles of 128 x {64,128} x 64 bytes are staged through LDS (rows padded to
// 80 bytes so the 16-lane row groups of ds_read_b128 hit distinct banks) and
// fed to v_mfma_i32_16x16x64_i8.  Within an MFMA the reduction index is just
// "byte b of lane group g", applied identically to A and B, so the exact sum
// does not depend on how the hardware orders k.
//
// Sums are exact: |sum| <= 131071 * 128^2 < 2^31 for every supported shape.
#include "iseg_common.h"

typedef int v4i __attribute__((ext_vector_type(4)));

namespace {

constexpr int BK = 64;        // reduction bytes per pipeline step
constexpr int ROW = 80;       // LDS row stride in bytes (64 + 16 pad)
constexpr int kMaxKred = 131071;
constexpr int64_t kWgradSplit = 131008;   // pixels per int32 partial (mult. of 64)

enum { MODE_FWD = 0, MODE_BWD = 1 };

struct IgemmArgs {
    const int8_t* src;            // NHWC [N, Hs, Ws, Ci]
    const int8_t* wmat;           // [Nout][Kred]
    int32_t* out;                 // [Mrows][Nout]
    unsigned long long* maxp;     // max |sum| (may be null)
    int64_t Mrows;
    int32_t Nout, Kred, Ci;
    int32_t Hs, Ws, Ho, Wo;
    int32_t R, S;
    int32_t sh, sw, ph, pw, dh, dw;
};

struct RowPix {
    int32_t n, oh, ow;
    bool ok;
};

__device__ __forceinline__ RowPix row_pix(const IgemmArgs& a, int64_t m)
{
    RowPix rp;
    rp.ok = m < a.Mrows;
    int64_t mm = rp.ok ? m : 0;
    int64_t hw = (int64_t)a.Ho * a.Wo;
    rp.n = (int32_t)(mm / hw);
    int32_t rem = (int32_t)(mm - (int64_t)rp.n * hw);
    rp.oh = rem / a.Wo;
    rp.ow = rem - rp.oh * a.Wo;
    return rp;
}

// source pixel of a row for tap (r,s); returns -1 if it contributes nothing
template <int MODE>
__device__ __forceinline__ int64_t src_pixel(const IgemmArgs& a, const RowPix& rp, int r, int s)
{
    int ih, iw;
    if (MODE == MODE_FWD) {
        ih = rp.oh * a.sh - a.ph + r * a.dh;
        iw = rp.ow * a.sw - a.pw + s * a.dw;
    } else {
        int nh = rp.oh + a.ph - r * a.dh;
        int nw = rp.ow + a.pw - s * a.dw;
        if (nh < 0 || nw < 0) return -1;
        ih = nh / a.sh;
        iw = nw / a.sw;
        if (ih * a.sh != nh || iw * a.sw != nw) return -1;
    }
    if (!rp.ok || ih < 0 || iw < 0 || ih >= a.Hs || iw >= a.Ws) return -1;
    return ((int64_t)rp.n * a.Hs + ih) * a.Ws + iw;
}

template <int MODE, bool VEC>
__device__ __forceinline__ int4 load_a_piece(const IgemmArgs& a, const RowPix& rp, int kk0)
{
    if (VEC) {
        if (kk0 >= a.Kred) return make_int4(0, 0, 0, 0);
        int tap = kk0 / a.Ci;
        int c0 = kk0 - tap * a.Ci;
        int r = tap / a.S, s = tap - (tap / a.S) * a.S;
        int64_t sp = src_pixel<MODE>(a, rp, r, s);
        if (sp < 0) return make_int4(0, 0, 0, 0);
        return *(const int4*)(a.src + sp * a.Ci + c0);
    } else {
        uint32_t w[4] = {0, 0, 0, 0};
        for (int b = 0; b < 16; b++) {
            int kk = kk0 + b;
            if (kk >= a.Kred) break;
            int tap = kk / a.Ci;
            int c = kk - tap * a.Ci;
            int r = tap / a.S, s = tap - (tap / a.S) * a.S;
            int64_t sp = src_pixel<MODE>(a, rp, r, s);
            if (sp >= 0) w[b >> 2] |= (uint32_t)(uint8_t)a.src[sp * a.Ci + c] << ((b & 3) * 8);
        }
        return make_int4((int)w[0], (int)w[1], (int)w[2], (int)w[3]);
    }
}

template <bool VEC>
__device__ __forceinline__ int4 load_b_piece(const IgemmArgs& a, int n, int kk0)
{
    if (n >= a.Nout || kk0 >= a.Kred) return make_int4(0, 0, 0, 0);
    const int8_t* p = a.wmat + (int64_t)n * a.Kred + kk0;
    if (VEC) return *(const int4*)p;
    uint32_t w[4] = {0, 0, 0, 0};
    for (int b = 0; b < 16 && kk0 + b < a.Kred; b++)
        w[b >> 2] |= (uint32_t)(uint8_t)p[b] << ((b & 3) * 8);
    return make_int4((int)w[0], (int)w[1], (int)w[2], (int)w[3]);
}

template <int MODE, bool VEC, int BM, int BN>
__global__ __launch_bounds__(256) void k_conv_igemm(IgemmArgs a)
{
    constexpr int PA = BM * 4 / 256;          // 16-byte A pieces per thread
    constexpr int PB = BN * 4 / 256;
    constexpr int WM = BM / 2, WN = BN / 2;   // wave tile (2 x 2 waves)
    constexpr int TM = WM / 16, TN = WN / 16;
    __shared__ __attribute__((aligned(16))) int8_t As[BM * ROW];
    __shared__ __attribute__((aligned(16))) int8_t Bs[BN * ROW];

    const int tid = threadIdx.x;
    const int64_t m0 = (int64_t)blockIdx.x * BM;
    const int n0 = blockIdx.y * BN;

    RowPix rp[PA];
#pragma unroll
    for (int j = 0; j < PA; j++) rp[j] = row_pix(a, m0 + ((tid + 256 * j) >> 2));

    const int nk = (a.Kred + BK - 1) / BK;
    int4 ra[PA], rb[PB];
#pragma unroll
    for (int j = 0; j < PA; j++) ra[j] = load_a_piece<MODE, VEC>(a, rp[j], ((tid + 256 * j) & 3) * 16);
#pragma unroll
    for (int j = 0; j < PB; j++) rb[j] = load_b_piece<VEC>(a, n0 + ((tid + 256 * j) >> 2), ((tid + 256 * j) & 3) * 16);

    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int lrow = lane & 15, lk = (lane >> 4) * 16;
    v4i acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; i++)
#pragma unroll
        for (int j = 0; j < TN; j++) acc[i][j] = (v4i){0, 0, 0, 0};

    for (int kb = 0; kb < nk; kb++) {
        __syncthreads();
#pragma unroll
        for (int j = 0; j < PA; j++) {
            int pi = tid + 256 * j;
            *(int4*)&As[(pi >> 2) * ROW + (pi & 3) * 16] = ra[j];
        }
#pragma unroll
        for (int j = 0; j < PB; j++) {
            int pi = tid + 256 * j;
            *(int4*)&Bs[(pi >> 2) * ROW + (pi & 3) * 16] = rb[j];
        }
        __syncthreads();
        if (kb + 1 < nk) {
            int kbase = (kb + 1) * BK;
#pragma unroll
            for (int j = 0; j < PA; j++)
                ra[j] = load_a_piece<MODE, VEC>(a, rp[j], kbase + ((tid + 256 * j) & 3) * 16);
#pragma unroll
            for (int j = 0; j < PB; j++)
                rb[j] = load_b_piece<VEC>(a, n0 + ((tid + 256 * j) >> 2), kbase + ((tid + 256 * j) & 3) * 16);
        }
        v4i fa[TM], fb[TN];
#pragma unroll
        for (int i = 0; i < TM; i++) fa[i] = *(const v4i*)&As[(wm * WM + i * 16 + lrow) * ROW + lk];
#pragma unroll
        for (int j = 0; j < TN; j++) fb[j] = *(const v4i*)&Bs[(wn * WN + j * 16 + lrow) * ROW + lk];
#pragma unroll
        for (int i = 0; i < TM; i++)
#pragma unroll
            for (int j = 0; j < TN; j++)
                acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[i], fb[j], acc[i][j], 0, 0, 0);
    }

    // epilogue: D[row = 4*(lane/16) + e][col = lane%16] of each 16x16 block
    uint64_t mx = 0;
#pragma unroll
    for (int i = 0; i < TM; i++)
#pragma unroll
        for (int j = 0; j < TN; j++) {
            int n = n0 + wn * WN + j * 16 + lrow;
#pragma unroll
            for (int e = 0; e < 4; e++) {
                int64_t m = m0 + wm * WM + i * 16 + (lane >> 4) * 4 + e;
                if (m < a.Mrows && n < a.Nout) {
                    int32_t v = acc[i][j][e];
                    a.out[m * a.Nout + n] = v;
                    uint64_t av = v < 0 ? (uint64_t)(-(int64_t)v) : (uint64_t)v;
                    mx = av > mx ? av : mx;
                }
            }
        }
    if (a.maxp) block_atomic_max_u64(mx, a.maxp);
}

template <int MODE>
int launch_igemm(const IgemmArgs& a, hipStream_t s)
{
    if (a.Mrows <= 0 || a.Nout <= 0) return ISEG_OK;
    bool vec = (a.Ci % 16) == 0 && (((uintptr_t)a.src | (uintptr_t)a.wmat) & 15) == 0;
    dim3 block(256);
    unsigned gx = (unsigned)ceil_div64(a.Mrows, 128);
    const int kid = MODE == MODE_FWD ? ISEG_KID_CONV_FWD : ISEG_KID_CONV_BWD_DATA;
    if (a.Nout > 64) {
        dim3 grid(gx, (unsigned)ceil_div64(a.Nout, 128));
        if (vec) ISEG_TIMED_LAUNCH(kid, s, (k_conv_igemm<MODE, true, 128, 128>), grid, block, 0, s, a);
        else ISEG_TIMED_LAUNCH(kid, s, (k_conv_igemm<MODE, false, 128, 128>), grid, block, 0, s, a);
    } else {
        dim3 grid(gx, 1);
        if (vec) ISEG_TIMED_LAUNCH(kid, s, (k_conv_igemm<MODE, true, 128, 64>), grid, block, 0, s, a);
        else ISEG_TIMED_LAUNCH(kid, s, (k_conv_igemm<MODE, false, 128, 64>), grid, block, 0, s, a);
    }
    return launch_ok();
}

// ---------------------------------------------------------------------------
// weights KRSC -> CRSK for the backward-data GEMM
// ---------------------------------------------------------------------------
__global__ void k_w_transpose(const int8_t* __restrict__ w, int8_t* __restrict__ wt,
                              int32_t K, int32_t RS, int32_t C)
{
    int64_t n = (int64_t)K * RS * C;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        // i indexes wt [c][rs][k]
        int32_t k = (int32_t)(i % K);
        int64_t t = i / K;
        int32_t rs = (int32_t)(t % RS);
        int32_t c = (int32_t)(t / RS);
        wt[i] = w[((int64_t)k * RS + rs) * C + c];
    }
}

__global__ void k_exp_sum(int32_t* out, const int32_t* a, const int32_t* b)
{
    *out = (a ? *a : 0) + (b ? *b : 0);
}

// ---------------------------------------------------------------------------
// backward-weight: G[k][(r,s,c)] = sum over pixels of dy[pix][k] * x[src(pix,r,s)][c]
// ---------------------------------------------------------------------------
struct WgradArgs {
    const int8_t* dy;        // [NPQ][K]
    const int8_t* x;         // [N,H,W,C]
    unsigned long long* acc; // int64 [K][RSC], accumulated atomically
    int64_t NPQ, pix_per_split;
    int32_t K, C, R, S, H, W, P, Q, RSC;
    int32_t sh, sw, ph, pw, dh, dw;
};

__device__ __forceinline__ uint32_t byte_of(uint32_t v, int c) { return (v >> (8 * c)) & 0xffu; }

// transpose of a 4x4 byte block: in[i] byte c -> out[c] byte i
__device__ __forceinline__ void transpose4x4(const uint32_t in[4], uint32_t out[4])
{
#pragma unroll
    for (int c = 0; c < 4; c++)
        out[c] = byte_of(in[0], c) | (byte_of(in[1], c) << 8) | (byte_of(in[2], c) << 16) |
                 (byte_of(in[3], c) << 24);
}

template <bool VEC, int BM, int BN>
__global__ __launch_bounds__(256) void k_conv_wgrad(WgradArgs a)
{
    constexpr int WM = BM / 2, WN = BN / 2;
    constexpr int TM = WM / 16, TN = WN / 16;
    constexpr int QA = BM / 64;   // 4x4 byte blocks per thread for the dy tile
    constexpr int QB = BN / 64;   // ... and for the x tile
    __shared__ __attribute__((aligned(16))) int8_t As[BM * ROW];   // [k][64 pixels]
    __shared__ __attribute__((aligned(16))) int8_t Bs[BN * ROW];   // [j][64 pixels]

    const int tid = threadIdx.x;
    const int j0 = blockIdx.x * BN;
    const int k0 = blockIdx.y * BM;
    const int64_t pbeg = (int64_t)blockIdx.z * a.pix_per_split;
    int64_t pend = pbeg + a.pix_per_split;
    if (pend > a.NPQ) pend = a.NPQ;
    const int64_t PQ = (int64_t)a.P * a.Q;

    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int lrow = lane & 15, lk = (lane >> 4) * 16;
    v4i acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; i++)
#pragma unroll
        for (int j = 0; j < TN; j++) acc[i][j] = (v4i){0, 0, 0, 0};

    for (int64_t pb = pbeg; pb < pend; pb += BK) {
        uint32_t ta[QA][4], tb[QB][4];
        // dy tile: 64 pixels x BM channels, 4x4 blocks (channel-group fastest)
#pragma unroll
        for (int q = 0; q < QA; q++) {
            int bi = tid + 256 * q;
            int cg = bi % (BM / 4), pg = bi / (BM / 4);
            uint32_t in[4];
#pragma unroll
            for (int i = 0; i < 4; i++) {
                int64_t pix = pb + pg * 4 + i;
                int kc = k0 + cg * 4;
                in[i] = 0;
                if (pix < pend) {
                    const int8_t* p = a.dy + pix * a.K + kc;
                    if (VEC) {
                        if (kc < a.K) in[i] = *(const uint32_t*)p;
                    } else {
                        for (int c = 0; c < 4; c++)
                            if (kc + c < a.K) in[i] |= (uint32_t)(uint8_t)p[c] << (8 * c);
                    }
                }
            }
            transpose4x4(in, ta[q]);
        }
        // x tile: 64 pixels x BN columns j = (r,s,c)
#pragma unroll
        for (int q = 0; q < QB; q++) {
            int bi = tid + 256 * q;
            int cg = bi % (BN / 4), pg = bi / (BN / 4);
            uint32_t in[4];
#pragma unroll
            for (int i = 0; i < 4; i++) {
                int64_t pix = pb + pg * 4 + i;
                in[i] = 0;
                if (pix >= pend) continue;
                int32_t n = (int32_t)(pix / PQ);
                int32_t rem = (int32_t)(pix - (int64_t)n * PQ);
                int32_t p = rem / a.Q, qq = rem - (rem / a.Q) * a.Q;
                for (int c = 0; c < 4; c++) {
                    int j = j0 + cg * 4 + c;
                    if (j >= a.RSC) break;
                    int tap = j / a.C, ch = j - (j / a.C) * a.C;
                    int r = tap / a.S, s = tap - (tap / a.S) * a.S;
                    int ih = p * a.sh - a.ph + r * a.dh, iw = qq * a.sw - a.pw + s * a.dw;
                    bool ok = ih >= 0 && iw >= 0 && ih < a.H && iw < a.W;
                    const int8_t* src = a.x + (((int64_t)n * a.H + ih) * a.W + iw) * a.C + ch;
                    if (VEC) {
                        // four consecutive channels of one tap
                        if (ok) in[i] = *(const uint32_t*)src;
                        break;
                    }
                    if (ok) in[i] |= (uint32_t)(uint8_t)*src << (8 * c);
                }
            }
            transpose4x4(in, tb[q]);
        }
        __syncthreads();
#pragma unroll
        for (int q = 0; q < QA; q++) {
            int bi = tid + 256 * q;
            int cg = bi % (BM / 4), pg = bi / (BM / 4);
#pragma unroll
            for (int c = 0; c < 4; c++) *(uint32_t*)&As[(cg * 4 + c) * ROW + pg * 4] = ta[q][c];
        }
#pragma unroll
        for (int q = 0; q < QB; q++) {
            int bi = tid + 256 * q;
            int cg = bi % (BN / 4), pg = bi / (BN / 4);
#pragma unroll
            for (int c = 0; c < 4; c++) *(uint32_t*)&Bs[(cg * 4 + c) * ROW + pg * 4] = tb[q][c];
        }
        __syncthreads();
        v4i fa[TM], fb[TN];
#pragma unroll
        for (int i = 0; i < TM; i++) fa[i] = *(const v4i*)&As[(wm * WM + i * 16 + lrow) * ROW + lk];
#pragma unroll
        for (int j = 0; j < TN; j++) fb[j] = *(const v4i*)&Bs[(wn * WN + j * 16 + lrow) * ROW + lk];
#pragma unroll
        for (int i = 0; i < TM; i++)
#pragma unroll
            for (int j = 0; j < TN; j++)
                acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[i], fb[j], acc[i][j], 0, 0, 0);
    }

#pragma unroll
    for (int i = 0; i < TM; i++)
#pragma unroll
        for (int j = 0; j < TN; j++) {
            int col = j0 + wn * WN + j * 16 + lrow;
#pragma unroll
            for (int e = 0; e < 4; e++) {
                int k = k0 + wm * WM + i * 16 + (lane >> 4) * 4 + e;
                int32_t v = acc[i][j][e];
                if (k < a.K && col < a.RSC && v != 0)
                    atomicAdd(&a.acc[(int64_t)k * a.RSC + col], (unsigned long long)(int64_t)v);
            }
        }
}

int launch_wgrad(WgradArgs a, hipStream_t s)
{
    if (a.NPQ <= 0) return ISEG_OK;
    bool vec = (a.C % 4) == 0 && (a.K % 4) == 0;
    constexpr int BM = 64, BN = 64;
    int64_t tiles = ceil_div64(a.K, BM) * ceil_div64(a.RSC, BN);
    int64_t splits = ceil_div64(2048, tiles);
    int64_t min_splits = ceil_div64(a.NPQ, kWgradSplit);
    int64_t max_splits = ceil_div64(a.NPQ, 64 * 4);
    if (splits > max_splits) splits = max_splits;
    if (splits < min_splits) splits = min_splits;
    if (splits > 65535) splits = 65535;
    int64_t pps = ceil_div64(ceil_div64(a.NPQ, splits), 64) * 64;
    if (pps > kWgradSplit) pps = kWgradSplit;
    a.pix_per_split = pps;
    splits = ceil_div64(a.NPQ, pps);
    dim3 grid((unsigned)ceil_div64(a.RSC, BN), (unsigned)ceil_div64(a.K, BM), (unsigned)splits);
    if (vec) ISEG_TIMED_LAUNCH(ISEG_KID_CONV_WGRAD, s, (k_conv_wgrad<true, BM, BN>), grid, dim3(256), 0, s, a);
    else ISEG_TIMED_LAUNCH(ISEG_KID_CONV_WGRAD, s, (k_conv_wgrad<false, BM, BN>), grid, dim3(256), 0, s, a);
    return launch_ok();
}

bool geom_ok(const iseg_conv_geom* g, int64_t* P, int64_t* Q)
{
    if (!g || g->N < 0 || g->H < 1 || g->W < 1 || g->C < 1 || g->K < 1 || g->R < 1 || g->S < 1)
        return false;
    if (g->stride_h < 1 || g->stride_w < 1 || g->dil_h < 1 || g->dil_w < 1 || g->pad_h < 0 ||
        g->pad_w < 0)
        return false;
    int64_t p = (g->H + 2 * g->pad_h - g->dil_h * (g->R - 1) - 1);
    int64_t q = (g->W + 2 * g->pad_w - g->dil_w * (g->S - 1) - 1);
    if (p < 0 || q < 0) return false;
    *P = p / g->stride_h + 1;
    *Q = q / g->stride_w + 1;
    if (g->H > (1 << 20) || g->W > (1 << 20) || g->C > (1 << 20) || g->K > (1 << 20)) return false;
    return true;
}

}  // namespace

// ---------------------------------------------------------------------------
// C ABI
// ---------------------------------------------------------------------------
extern "C" size_t iseg_conv_fwd_ws(const iseg_conv_geom* g, int32_t out_mode)
{
    int64_t P, Q;
    if (!geom_ok(g, &P, &Q)) return 0;
    size_t s = 256;
    if (out_mode == ISEG_OUT_Q8) s += align256((size_t)(g->N * P * Q * g->K) * 4);
    return s;
}

extern "C" int iseg_conv_fwd(const int8_t* x, const int32_t* x_exp, const int8_t* w, const int32_t* w_exp,
                             const iseg_conv_geom* g, int32_t out_mode, void* y, int32_t* y_exp,
                             void* ws, size_t ws_bytes, int32_t* dev_status, hipStream_t stream)
{
    (void)dev_status;
    int64_t P, Q;
    if (!geom_ok(g, &P, &Q)) return ISEG_ERR_SHAPE;
    if (out_mode != ISEG_OUT_Q8 && out_mode != ISEG_OUT_RAW) return ISEG_ERR_ARG;
    if (!x_exp || !w_exp || !y_exp || (g->N > 0 && (!x || !w || !y))) return ISEG_ERR_ARG;
    if (g->C * g->R * g->S > kMaxKred) return ISEG_ERR_UNSUPPORTED;
    if (!ws || ws_bytes < iseg_conv_fwd_ws(g, out_mode)) return ISEG_ERR_WORKSPACE;
    unsigned long long* maxp = (unsigned long long*)ws;
    int32_t* acc = out_mode == ISEG_OUT_Q8 ? (int32_t*)((char*)ws + 256) : (int32_t*)y;
    int rc = launch_fill_u32(maxp, 2, 0, stream);
    if (rc) return rc;
    IgemmArgs a;
    a.src = x; a.wmat = w; a.out = acc; a.maxp = out_mode == ISEG_OUT_Q8 ? maxp : nullptr;
    a.Mrows = g->N * P * Q;
    a.Nout = (int32_t)g->K; a.Kred = (int32_t)(g->C * g->R * g->S); a.Ci = (int32_t)g->C;
    a.Hs = (int32_t)g->H; a.Ws = (int32_t)g->W; a.Ho = (int32_t)P; a.Wo = (int32_t)Q;
    a.R = (int32_t)g->R; a.S = (int32_t)g->S;
    a.sh = g->stride_h; a.sw = g->stride_w; a.ph = g->pad_h; a.pw = g->pad_w;
    a.dh = g->dil_h; a.dw = g->dil_w;
    if ((rc = launch_igemm<MODE_FWD>(a, stream))) return rc;
    if (out_mode == ISEG_OUT_RAW) {
        hipLaunchKernelGGL(k_exp_sum, dim3(1), dim3(1), 0, stream, y_exp, x_exp, w_exp);
        return launch_ok();
    }
    return launch_requant_apply(acc, ISEG_I32, a.Mrows * a.Nout, x_exp, w_exp, 0, 8, 0, 1,
                                0, 0, 0, ISEG_I8, y, y_exp, maxp, stream);
}

extern "C" size_t iseg_conv_bwd_data_ws(const iseg_conv_geom* g, int32_t out_mode)
{
    int64_t P, Q;
    if (!geom_ok(g, &P, &Q)) return 0;
    size_t s = 256 + align256((size_t)(g->K * g->R * g->S * g->C));
    if (out_mode == ISEG_OUT_Q8) s += align256((size_t)(g->N * g->H * g->W * g->C) * 4);
    return s;
}

extern "C" int iseg_conv_bwd_data(const int8_t* dy, const int32_t* dy_exp, const int8_t* w,
                                  const int32_t* w_exp, const iseg_conv_geom* g, int32_t out_mode,
                                  void* dx, int32_t* dx_exp, void* ws, size_t ws_bytes,
                                  int32_t* dev_status, hipStream_t stream)
{
    (void)dev_status;
    int64_t P, Q;
    if (!geom_ok(g, &P, &Q)) return ISEG_ERR_SHAPE;
    if (out_mode != ISEG_OUT_Q8 && out_mode != ISEG_OUT_RAW) return ISEG_ERR_ARG;
    if (!dy_exp || !w_exp || !dx_exp || (g->N > 0 && (!dy || !w || !dx))) return ISEG_ERR_ARG;
    if (g->K * g->R * g->S > kMaxKred) return ISEG_ERR_UNSUPPORTED;
    if (!ws || ws_bytes < iseg_conv_bwd_data_ws(g, out_mode)) return ISEG_ERR_WORKSPACE;
    unsigned long long* maxp = (unsigned long long*)ws;
    int8_t* wt = (int8_t*)ws + 256;
    size_t wt_bytes = align256((size_t)(g->K * g->R * g->S * g->C));
    int32_t* acc = out_mode == ISEG_OUT_Q8 ? (int32_t*)((char*)ws + 256 + wt_bytes) : (int32_t*)dx;
    int rc = launch_fill_u32(maxp, 2, 0, stream);
    if (rc) return rc;
    int64_t nw = g->K * g->R * g->S * g->C;
    hipLaunchKernelGGL(k_w_transpose, dim3(grid_for(nw, 256, 4096)), dim3(256), 0, stream, w, wt,
                       (int32_t)g->K, (int32_t)(g->R * g->S), (int32_t)g->C);
    if ((rc = launch_ok())) return rc;
    IgemmArgs a;
    a.src = dy; a.wmat = wt; a.out = acc; a.maxp = out_mode == ISEG_OUT_Q8 ? maxp : nullptr;
    a.Mrows = g->N * g->H * g->W;
    a.Nout = (int32_t)g->C; a.Kred = (int32_t)(g->K * g->R * g->S); a.Ci = (int32_t)g->K;
    a.Hs = (int32_t)P; a.Ws = (int32_t)Q; a.Ho = (int32_t)g->H; a.Wo = (int32_t)g->W;
    a.R = (int32_t)g->R; a.S = (int32_t)g->S;
    a.sh = g->stride_h; a.sw = g->stride_w; a.ph = g->pad_h; a.pw = g->pad_w;
    a.dh = g->dil_h; a.dw = g->dil_w;
    if ((rc = launch_igemm<MODE_BWD>(a, stream))) return rc;
    if (out_mode == ISEG_OUT_RAW) {
        hipLaunchKernelGGL(k_exp_sum, dim3(1), dim3(1), 0, stream, dx_exp, dy_exp, w_exp);
        return launch_ok();
    }
    return launch_requant_apply(acc, ISEG_I32, a.Mrows * a.Nout, dy_exp, w_exp, 0, 8, 0, 1,
                                0, 0, 0, ISEG_I8, dx, dx_exp, maxp, stream);
}

extern "C" size_t iseg_conv_bwd_weight_ws(const iseg_conv_geom* g, int32_t g_mode)
{
    int64_t P, Q;
    if (!geom_ok(g, &P, &Q)) return 0;
    (void)g_mode;
    return 256 + align256((size_t)(g->K * g->R * g->S * g->C) * 8);
}

extern "C" int iseg_conv_bwd_weight(const int8_t* dy, const int32_t* dy_exp, const int8_t* x,
                                    const int32_t* x_exp, const iseg_conv_geom* g, int32_t g_mode,
                                    int32_t bits, uint64_t seed, uint32_t tensor_id, uint32_t step,
                                    void* dw, int32_t* dw_exp, void* ws, size_t ws_bytes,
                                    int32_t* dev_status, hipStream_t stream)
{
    int64_t P, Q;
    if (!geom_ok(g, &P, &Q)) return ISEG_ERR_SHAPE;
    if (g_mode != ISEG_G_KEEP && g_mode != ISEG_G_DROP && g_mode != ISEG_G_RAW) return ISEG_ERR_ARG;
    if (g_mode != ISEG_G_RAW && (bits < 2 || bits > 8)) return ISEG_ERR_ARG;
    if (!dy_exp || !x_exp || !dw_exp || !dw || (g->N > 0 && (!dy || !x))) return ISEG_ERR_ARG;
    if (!ws || ws_bytes < iseg_conv_bwd_weight_ws(g, g_mode)) return ISEG_ERR_WORKSPACE;
    unsigned long long* maxp = (unsigned long long*)ws;
    int64_t nw = g->K * g->R * g->S * g->C;
    unsigned long long* acc = g_mode == ISEG_G_RAW ? (unsigned long long*)dw
                                                   : (unsigned long long*)((char*)ws + 256);
    int rc = launch_fill_u32(maxp, 2, 0, stream);
    if (!rc) rc = launch_fill_u32(acc, nw * 2, 0, stream);
    if (rc) return rc;
    WgradArgs a;
    a.dy = dy; a.x = x; a.acc = acc;
    a.NPQ = g->N * P * Q; a.pix_per_split = 0;
    a.K = (int32_t)g->K; a.C = (int32_t)g->C; a.R = (int32_t)g->R; a.S = (int32_t)g->S;
    a.H = (int32_t)g->H; a.W = (int32_t)g->W; a.P = (int32_t)P; a.Q = (int32_t)Q;
    a.RSC = (int32_t)(g->R * g->S * g->C);
    a.sh = g->stride_h; a.sw = g->stride_w; a.ph = g->pad_h; a.pw = g->pad_w;
    a.dh = g->dil_h; a.dw = g->dil_w;
    if ((rc = launch_wgrad(a, stream))) return rc;
    if (g_mode == ISEG_G_RAW) {
        hipLaunchKernelGGL(k_exp_sum, dim3(1), dim3(1), 0, stream, dw_exp, dy_exp, x_exp);
        return launch_ok();
    }
    if ((rc = launch_absmax(acc, ISEG_I64, nw, maxp, dev_status, stream))) return rc;
    int keep = g_mode == ISEG_G_KEEP;
    return launch_requant_apply(acc, ISEG_I64, nw, keep ? dy_exp : nullptr, keep ? x_exp : nullptr,
                                0, bits, 1, keep, seed, tensor_id, step, ISEG_I8, dw, dw_exp,
                                maxp, stream);
}
