// loss.hip -- the float region of a segmentation training step on gfx950.
//
// The int8 logits [N,h,w,K] (one power-of-two exponent) are upsampled
// bilinearly to the label size [N,H,W] (half-pixel centres: source coordinate
// (o + 1/2) n_in / n_out - 1/2 clamped at 0, upper neighbour clamped at the
// edge), scored by the pixel-wise softmax cross-entropy (mean over the N H W
// pixels), differentiated, taken back through the adjoint of the upsampling,
// and quantized by SQ to the int8 error E1 at the logits (Eq. 4 / Eq. 16: the
// one float -> integer crossing of the dataflow).
//
// Float64 throughout, so that the integer codes decided at the end agree with
// a float64 reference except where a value sits within ~1e-14 relative of a
// rounding boundary.  Deterministic: every sum runs in a fixed order.
//   k_ce_rows   one block per hi-res row: softmax per pixel (one wave per
//               pixel, lanes over classes), gradient staged in LDS for 16
//               pixels, folded into the row's column adjoint held in LDS;
//               writes the row adjoint [N,H,w,K] and the row's loss
//   k_ce_cols   one lane per low-res element: the row adjoint folded over
//               the hi-res rows that read it -> gradient, |.| max partials
//   k_ce_quant  SQ codes and exponent; block 0 also forms the mean loss
#include <math.h>

#include "iseg_common.h"

namespace {

struct CeArgs {
    const int8_t* logits;
    const int32_t* logit_exp;
    const uint8_t* labels;
    int32_t N, h, w, K, H, W;
    double* gx;          // [N, H, w, K]
    double* row_loss;    // [N * H]
    double* grad;        // [N, h, w, K]
    uint64_t* part;      // |grad| max partials
    int32_t* status;
};

__device__ __forceinline__ void src_coord(int o, int n_in, int n_out, int& i0, int& i1, double& lam)
{
    double src = ((double)o + 0.5) * (double)n_in / (double)n_out - 0.5;
    if (src < 0.0) src = 0.0;
    i0 = (int)floor(src);
    i1 = i0 + 1 < n_in ? i0 + 1 : n_in - 1;
    lam = src - (double)i0;
}

__device__ __forceinline__ double wave_max_f64(double v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o, 64));
    return v;
}

__device__ __forceinline__ double wave_sum_f64(double v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

constexpr int kChunk = 16;     // pixels whose gradient is staged in LDS at a time

template <int KT>
__global__ __launch_bounds__(256) void k_ce_rows(CeArgs a)
{
    extern __shared__ __align__(16) char smem[];
    __shared__ int cj0[kChunk], cj1[kChunk];
    __shared__ double cw0[kChunk], cw1[kChunk];
    __shared__ double wloss[4];
    const int y = blockIdx.x, n = blockIdx.y;
    const int K = a.K, w = a.w, wk = a.w * a.K;
    int8_t* L0 = (int8_t*)smem;                                   // [w][K] top source row
    int8_t* L1 = L0 + wk;                                         // [w][K] bottom source row
    double* gbuf = (double*)(smem + ((2 * wk + 15) & ~15));       // [kChunk][K]
    double* gx = gbuf + kChunk * K;                               // [w][K]

    int i0, i1;
    double ly;
    src_coord(y, a.h, a.H, i0, i1, ly);
    const double wy0 = 1.0 - ly, wy1 = ly;
    const int8_t* r0 = a.logits + ((int64_t)n * a.h + i0) * wk;
    const int8_t* r1 = a.logits + ((int64_t)n * a.h + i1) * wk;
    for (int t = threadIdx.x; t < wk; t += blockDim.x) {
        L0[t] = r0[t];
        L1[t] = r1[t];
        gx[t] = 0.0;
    }
    const double scale = ldexp(1.0, *a.logit_exp);
    const double P = (double)a.N * (double)a.H * (double)a.W;
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const uint8_t* lab_row = a.labels + ((int64_t)n * a.H + y) * a.W;
    double lsum = 0.0;
    bool bad_label = false;
    __syncthreads();
    for (int x0 = 0; x0 < a.W; x0 += kChunk) {
        const int npx = a.W - x0 < kChunk ? a.W - x0 : kChunk;
        if (threadIdx.x < npx) {
            int j0, j1;
            double lx;
            src_coord(x0 + threadIdx.x, w, a.W, j0, j1, lx);
            cj0[threadIdx.x] = j0;
            cj1[threadIdx.x] = j1;
            cw0[threadIdx.x] = 1.0 - lx;
            cw1[threadIdx.x] = lx;
        }
        __syncthreads();
        // softmax of each pixel: one wave per pixel, lane k + 64 t holds class k + 64 t
        for (int pi = wv; pi < npx; pi += 4) {
            const int j0 = cj0[pi], j1 = cj1[pi];
            const double wx0 = cw0[pi], wx1 = cw1[pi];
            const int lab = lab_row[x0 + pi];
            bad_label |= lab >= K;
            double l[KT];
            double m = -INFINITY;
#pragma unroll
            for (int t = 0; t < KT; t++) {
                const int k = lane + 64 * t;
                if (k < K) {
                    const double top = wx0 * (double)L0[j0 * K + k] + wx1 * (double)L0[j1 * K + k];
                    const double bot = wx0 * (double)L1[j0 * K + k] + wx1 * (double)L1[j1 * K + k];
                    l[t] = (wy0 * top + wy1 * bot) * scale;
                    m = fmax(m, l[t]);
                } else {
                    l[t] = 0.0;
                }
            }
            m = wave_max_f64(m);
            double e[KT];
            double s = 0.0, ll = 0.0;
#pragma unroll
            for (int t = 0; t < KT; t++) {
                const int k = lane + 64 * t;
                e[t] = k < K ? exp(l[t] - m) : 0.0;
                s += e[t];
                if (k == lab) ll = l[t];
            }
            s = wave_sum_f64(s);
            ll = wave_sum_f64(ll);                 // one lane holds the label's logit
#pragma unroll
            for (int t = 0; t < KT; t++) {
                const int k = lane + 64 * t;
                if (k < K) gbuf[pi * K + k] = (e[t] / s - (k == lab ? 1.0 : 0.0)) / P;
            }
            if (lane == 0) lsum += log(s) + m - ll;
        }
        __syncthreads();
        // fold the chunk into the columns it touches, pixels in ascending order
        const int jlo = cj0[0], jhi = cj1[npx - 1];
        const int ncol = jhi - jlo + 1;
        for (int t = threadIdx.x; t < ncol * K; t += blockDim.x) {
            const int j = jlo + t / K, k = t % K;
            double acc = gx[j * K + k];
            for (int pi = 0; pi < npx; pi++) {
                double wgt = 0.0;
                if (cj0[pi] == j) wgt += cw0[pi];
                if (cj1[pi] == j) wgt += cw1[pi];
                if (wgt != 0.0) acc += wgt * gbuf[pi * K + k];
            }
            gx[j * K + k] = acc;
        }
        __syncthreads();
    }
    double* out = a.gx + ((int64_t)n * a.H + y) * wk;
    for (int t = threadIdx.x; t < wk; t += blockDim.x) out[t] = gx[t];
    if (lane == 0) wloss[wv] = lsum;
    if (bad_label && lane == 0) set_status(a.status, ISEG_DEV_RANGE);
    __syncthreads();
    if (threadIdx.x == 0) a.row_loss[(int64_t)n * a.H + y] = ((wloss[0] + wloss[1]) + wloss[2]) + wloss[3];
}

// grad[n,i,j,k] = sum over hi-res rows y of Ay[y,i] gx[n,y,j,k], y ascending
__global__ __launch_bounds__(256) void k_ce_cols(CeArgs a)
{
    const int64_t total = (int64_t)a.N * a.h * a.w * a.K;
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    uint64_t m = 0;
    if (e < total) {
        const int64_t wk = (int64_t)a.w * a.K;
        const int64_t jk = e % wk;
        const int64_t ni = e / wk;
        const int i = (int)(ni % a.h);
        const int n = (int)(ni / a.h);
        const double sc = (double)a.H / (double)a.h;
        int ylo = (int)floor(((double)i - 0.5) * sc - 0.5) - 1;
        int yhi = (int)ceil(((double)i + 1.5) * sc - 0.5) + 1;
        ylo = ylo < 0 ? 0 : ylo;
        yhi = yhi > a.H - 1 ? a.H - 1 : yhi;
        double acc = 0.0;
        const double* col = a.gx + (int64_t)n * a.H * wk + jk;
        for (int y = ylo; y <= yhi; y++) {
            int i0, i1;
            double ly;
            src_coord(y, a.h, a.H, i0, i1, ly);
            double wgt = 0.0;
            if (i0 == i) wgt += 1.0 - ly;
            if (i1 == i) wgt += ly;
            if (wgt != 0.0) acc += wgt * col[(int64_t)y * wk];
        }
        a.grad[e] = acc;
        m = (uint64_t)__double_as_longlong(acc) & 0x7fffffffffffffffull;
    }
    block_store_max_u64(m, a.part);
}

// smallest e with |v| < 2^e for the positive double with bits mb (frexp's exponent)
__device__ __forceinline__ int frexp_exp_bits64(uint64_t mb)
{
    const int E = (int)(mb >> 52);
    const uint64_t man = mb & 0xfffffffffffffull;
    if (E == 0) return bitlen_u64(man) - 1074;
    return E - 1022;
}

__global__ __launch_bounds__(256) void k_ce_quant(CeArgs a, const unsigned long long* maxp, int bits,
                                                  int8_t* __restrict__ err, int32_t* err_exp, double* loss)
{
    const uint64_t mb = *maxp;
    const int b = mb ? frexp_exp_bits64(mb) : 0;
    const int64_t total = (int64_t)a.N * a.h * a.w * a.K;
    if (blockIdx.x == 0) {
        if (threadIdx.x == 0) *err_exp = b + 1 - bits;
        // mean loss: row losses summed in a fixed tree order
        __shared__ double red[256];
        double s = 0.0;
        const int64_t rows = (int64_t)a.N * a.H;
        for (int64_t r = threadIdx.x; r < rows; r += blockDim.x) s += a.row_loss[r];
        red[threadIdx.x] = s;
        __syncthreads();
        for (int o = 128; o > 0; o >>= 1) {
            if ((int)threadIdx.x < o) red[threadIdx.x] += red[threadIdx.x + o];
            __syncthreads();
        }
        if (threadIdx.x == 0 && loss) *loss = red[0] / ((double)a.N * (double)a.H * (double)a.W);
    }
    const int sh = bits - 1 - b;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        const double v = ldexp(a.grad[e], sh);      // a power-of-two scale: exact
        const double fl = floor(v);
        const double nf = fl + (v - fl >= 0.5 ? 1.0 : 0.0);
        err[e] = (int8_t)clamp_k((int64_t)nf, bits);
    }
}

template <int KT>
int launch_rows(const CeArgs& a, size_t lds, hipStream_t s)
{
    if (hipFuncSetAttribute((const void*)k_ce_rows<KT>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) !=
        hipSuccess)
        return ISEG_ERR_DEVICE;
    hipLaunchKernelGGL(k_ce_rows<KT>, dim3((unsigned)a.H, (unsigned)a.N), dim3(256), lds, s, a);
    return launch_ok();
}

size_t rows_lds(int64_t w, int64_t K)
{
    return (size_t)((2 * w * K + 15) & ~(int64_t)15) + (size_t)(kChunk * K + w * K) * 8;
}

}  // namespace

extern "C" size_t iseg_softmax_ce_ws(int64_t N, int64_t h, int64_t w, int64_t K, int64_t H, int64_t W)
{
    (void)W;
    const int64_t nlow = N * h * w * K;
    return 256 + align256((size_t)(N * H * w * K) * 8) + align256((size_t)(N * H) * 8) +
           align256((size_t)nlow * 8) + align256((size_t)ceil_div64(nlow, 256) * 8);
}

extern "C" int iseg_softmax_ce(const int8_t* logits, const int32_t* logit_exp, const uint8_t* labels, int64_t N,
                               int64_t h, int64_t w, int64_t K, int64_t H, int64_t W, int32_t bits, double* loss,
                               double* grad, int8_t* err, int32_t* err_exp, void* ws, size_t ws_bytes,
                               int32_t* dev_status, hipStream_t stream)
{
    if (N < 1 || h < 1 || w < 1 || K < 1 || H < h || W < w || bits < 2 || bits > 8) return ISEG_ERR_ARG;
    if (!logits || !logit_exp || !labels || !err || !err_exp) return ISEG_ERR_ARG;
    if (K > 256 || H > 65535 || N > 65535 || rows_lds(w, K) > 150 * 1024) return ISEG_ERR_UNSUPPORTED;
    if (!ws || ws_bytes < iseg_softmax_ce_ws(N, h, w, K, H, W)) return ISEG_ERR_WORKSPACE;
    CeArgs a{};
    a.logits = logits; a.logit_exp = logit_exp; a.labels = labels;
    a.N = (int32_t)N; a.h = (int32_t)h; a.w = (int32_t)w; a.K = (int32_t)K; a.H = (int32_t)H; a.W = (int32_t)W;
    a.status = dev_status;
    char* p = (char*)ws;
    unsigned long long* maxp = (unsigned long long*)p;
    p += 256;
    a.gx = (double*)p;
    p += align256((size_t)(N * H * w * K) * 8);
    a.row_loss = (double*)p;
    p += align256((size_t)(N * H) * 8);
    double* gws = (double*)p;
    p += align256((size_t)(N * h * w * K) * 8);
    a.part = (uint64_t*)p;
    a.grad = grad ? grad : gws;
    const int64_t nlow = N * h * w * K;
    const size_t lds = rows_lds(w, K);
    const int kt = (int)((K + 63) / 64);
    int rc = kt == 1 ? launch_rows<1>(a, lds, stream)
           : kt == 2 ? launch_rows<2>(a, lds, stream)
           : kt == 3 ? launch_rows<3>(a, lds, stream)
                     : launch_rows<4>(a, lds, stream);
    if (rc) return rc;
    const unsigned nb = (unsigned)ceil_div64(nlow, 256);
    hipLaunchKernelGGL(k_ce_cols, dim3(nb), dim3(256), 0, stream, a);
    if ((rc = launch_ok())) return rc;
    if ((rc = launch_reduce_max(a.part, nb, maxp, stream))) return rc;
    hipLaunchKernelGGL(k_ce_quant, dim3(grid_for(nlow, 256, 2048)), dim3(256), 0, stream, a,
                       (const unsigned long long*)maxp, (int)bits, err, err_exp, loss);
    return launch_ok();
}
