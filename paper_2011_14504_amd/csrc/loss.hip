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
//   k_ce_cells    one wave per bilinear cell (a run of output rows that read
//                 the same two source rows x a run of columns): softmax of each
//                 pixel with lanes over classes, the gradient folded into the
//                 cell's four source corners, the cell's loss
//   k_ce_combine  one block per low-res row: the corner sums of every cell
//                 touching each low-res element, in cell order -> gradient
//   k_ce_quant    SQ codes and exponent; block 0 also forms the mean loss
#include <math.h>

#include "iseg_common.h"

namespace {

// the logit exponents the region accepts: |logit| < 128, so every exp() of a
// difference of (bilinear mixes of) logits stays a normal finite double
constexpr int kLogitExpMin = -1000, kLogitExpMax = 0;
__device__ __forceinline__ bool logit_exp_ok(int32_t e) { return e >= kLogitExpMin && e <= kLogitExpMax; }


// 64-bit value moved across lanes by a DPP control (both 32-bit halves)
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v)
{
    const long long b = __double_as_longlong(v);
    const int lo = __builtin_amdgcn_mov_dpp((int)b, CTRL, 0xF, 0xF, false);
    const int hi = __builtin_amdgcn_mov_dpp((int)(b >> 32), CTRL, 0xF, 0xF, false);
    return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
}

__device__ __forceinline__ double readlane_f64(double v, int l)
{
    const long long b = __double_as_longlong(v);
    const int lo = __builtin_amdgcn_readlane((int)b, l);
    const int hi = __builtin_amdgcn_readlane((int)(b >> 32), l);
    return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
}

// Wave-wide sum / max, the same value in every lane: within each row of 16
// lanes by DPP steps whose pairs are symmetric (quad swaps, half-row and row
// mirrors), then the four row results added in a fixed order.
__device__ __forceinline__ double wave_sum_f64(double v)
{
    v += dpp_f64<0xB1>(v);      // quad_perm [1,0,3,2]
    v += dpp_f64<0x4E>(v);      // quad_perm [2,3,0,1]
    v += dpp_f64<0x141>(v);     // row_half_mirror
    v += dpp_f64<0x140>(v);     // row_mirror
    return (readlane_f64(v, 0) + readlane_f64(v, 16)) + (readlane_f64(v, 32) + readlane_f64(v, 48));
}

__device__ __forceinline__ double wave_max_f64(double v)
{
    v = fmax(v, dpp_f64<0xB1>(v));
    v = fmax(v, dpp_f64<0x4E>(v));
    v = fmax(v, dpp_f64<0x141>(v));
    v = fmax(v, dpp_f64<0x140>(v));
    return fmax(fmax(readlane_f64(v, 0), readlane_f64(v, 16)), fmax(readlane_f64(v, 32), readlane_f64(v, 48)));
}

// ---------------------------------------------------------------------------
// Runs: maximal ranges of output coordinates that read the same two source
// positions (i0, i1) with the same clamping, so that the interpolation weight
// is affine in the coordinate inside a run.  A cell is (row run) x (column
// run): its logits are bilinear in (x, y), so exp(l - m) follows a 2-D
// multiplicative recurrence: exp at one corner, the x-step ratio, the y-step
// ratio and the change of the x-step per row (4 exps per class and cell).
// ---------------------------------------------------------------------------
constexpr int kMaxRuns = 136;

struct Run {
    int16_t start, len, i0, i1;
};

struct CeCellArgs {
    const int8_t* logits;
    const int32_t* logit_exp;
    const uint8_t* labels;
    int32_t N, h, w, K, H, W;
    int32_t nry, nrx;
    Run ry[kMaxRuns];
    Run rx[kMaxRuns];
    double* cell;        // [N][nry][nrx][4][K]: corner sums (i0,j0),(i0,j1),(i1,j0),(i1,j1)
    double* cell_loss;   // [N][nry][nrx]
    double* grad;        // [N][h][w][K]
    uint64_t* part;      // |grad| max partials, one per combine block
    int32_t* status;
};

__host__ __device__ __forceinline__ void src_coord_hd(int o, int n_in, int n_out, int& i0, int& i1, double& lam,
                                                       bool& clamped)
{
    double src = ((double)o + 0.5) * (double)n_in / (double)n_out - 0.5;
    clamped = src < 0.0;
    if (clamped) src = 0.0;
    i0 = (int)floor(src);
    i1 = i0 + 1 < n_in ? i0 + 1 : n_in - 1;
    lam = src - (double)i0;
}

// host: run table of one axis; returns the count, or -1 above kMaxRuns
static int make_runs(int n_in, int n_out, Run* runs)
{
    int n = 0, pi0 = -1, pi1 = -1;
    bool pcl = false;
    for (int o = 0; o < n_out; o++) {
        int i0, i1;
        double lam;
        bool cl;
        src_coord_hd(o, n_in, n_out, i0, i1, lam, cl);
        if (o == 0 || i0 != pi0 || i1 != pi1 || cl != pcl) {
            if (n == kMaxRuns) return -1;
            runs[n].start = (int16_t)o;
            runs[n].len = 0;
            runs[n].i0 = (int16_t)i0;
            runs[n].i1 = (int16_t)i1;
            n++;
        }
        runs[n - 1].len++;
        pi0 = i0;
        pi1 = i1;
        pcl = cl;
    }
    return n;
}

__device__ __forceinline__ double interp(double a00, double a01, double a10, double a11, double wx0, double wx1,
                                         double wy0, double wy1, double scale)
{
    const double top = wx0 * a00 + wx1 * a01;
    const double bot = wx0 * a10 + wx1 * a11;
    return (wy0 * top + wy1 * bot) * scale;
}

// one block per cell, its rows split over the 4 waves: softmax of every pixel
// (lanes over classes), the gradient folded into the cell's four low-res
// corners (x first within a row, then the row weights), the cell's loss; the
// waves' corner sums are added in wave order
constexpr int kCellWaves = 4;
constexpr int kMaxRunLen = 256;
constexpr int kLabBuf = 1024;

template <int KT>
__global__ __launch_bounds__(256) void k_ce_cells(const CeCellArgs a)
{
    extern __shared__ __align__(16) char smem[];
    __shared__ double wxs[kMaxRunLen];                     // column weight lambda_x per pixel of the run
    __shared__ double wl[kCellWaves];
    __shared__ uint8_t labs[kCellWaves][kLabBuf];          // each wave's labels, a chunk of rows at a time
    const int n = blockIdx.z, sy = blockIdx.y, sx = blockIdx.x;
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int K = a.K, wk = a.w * a.K;
    const Run ry = a.ry[sy], rx = a.rx[sx];
    const int j0 = rx.i0, j1 = rx.i1;
    // the four corner columns of both source rows, and the reduction buffer
    int8_t* C0 = (int8_t*)smem;                            // [4][K]: (i0,j0) (i0,j1) (i1,j0) (i1,j1)
    double* red = (double*)(smem + ((4 * K + 15) & ~15));  // [waves][4][K]
    const int8_t* r0 = a.logits + ((int64_t)n * a.h + ry.i0) * wk;
    const int8_t* r1 = a.logits + ((int64_t)n * a.h + ry.i1) * wk;
    for (int t = threadIdx.x; t < K; t += blockDim.x) {
        C0[t] = r0[j0 * K + t];
        C0[K + t] = r0[j1 * K + t];
        C0[2 * K + t] = r1[j0 * K + t];
        C0[3 * K + t] = r1[j1 * K + t];
    }
    for (int c = threadIdx.x; c < rx.len; c += blockDim.x) {
        int e0, e1;
        bool ecl;
        double lx;
        src_coord_hd(rx.start + c, a.w, a.W, e0, e1, lx, ecl);
        wxs[c] = lx;
    }
    __syncthreads();
    // outside the documented range the outputs are discarded (k_ce_quant)
    const double scale = logit_exp_ok(*a.logit_exp) ? ldexp(1.0, *a.logit_exp) : 0.0;
    const double invP = 1.0 / ((double)a.N * (double)a.H * (double)a.W);

    double c00[KT], c01[KT], c10[KT], c11[KT];
    double m = -INFINITY;
#pragma unroll
    for (int t = 0; t < KT; t++) {
        const int k = lane + 64 * t;
        if (k < K) {
            c00[t] = C0[k];
            c01[t] = C0[K + k];
            c10[t] = C0[2 * K + k];
            c11[t] = C0[3 * K + k];
            m = fmax(m, fmax(fmax(c00[t], c01[t]), fmax(c10[t], c11[t])) * scale);
        } else {
            c00[t] = c01[t] = c10[t] = c11[t] = 0.0;
        }
    }
    m = wave_max_f64(m);

    // this wave's rows, and the weights at its first two rows / the run's first two columns
    const int rc = (ry.len + kCellWaves - 1) / kCellWaves;
    const int rbeg = wv * rc;
    const int rend = rbeg + rc < ry.len ? rbeg + rc : ry.len;
    double G00[KT], G01[KT], G10[KT], G11[KT];
#pragma unroll
    for (int t = 0; t < KT; t++) G00[t] = G01[t] = G10[t] = G11[t] = 0.0;
    double lsum = 0.0, luni = 0.0, llab = 0.0, sv = 1.0;
    int pc = 0;
    bool bad = false;
    if (rbeg < rend) {
        int d0, d1;
        bool dcl;
        double ly0, ly1;
        const double lx0 = wxs[0], lx1 = wxs[rx.len > 1 ? 1 : 0];
        src_coord_hd(ry.start + rbeg, a.h, a.H, d0, d1, ly0, dcl);
        src_coord_hd(ry.start + rbeg + (rend - rbeg > 1 ? 1 : 0), a.h, a.H, d0, d1, ly1, dcl);
        double Er[KT], Rr[KT], Qy[KT], Tx[KT];
#pragma unroll
        for (int t = 0; t < KT; t++) {
            const double l00 = interp(c00[t], c01[t], c10[t], c11[t], 1.0 - lx0, lx0, 1.0 - ly0, ly0, scale);
            const double l10 = interp(c00[t], c01[t], c10[t], c11[t], 1.0 - lx1, lx1, 1.0 - ly0, ly0, scale);
            const double l01 = interp(c00[t], c01[t], c10[t], c11[t], 1.0 - lx0, lx0, 1.0 - ly1, ly1, scale);
            const double l11 = interp(c00[t], c01[t], c10[t], c11[t], 1.0 - lx1, lx1, 1.0 - ly1, ly1, scale);
            const bool on = lane + 64 * t < K;
            Er[t] = on ? exp(l00 - m) : 0.0;
            Rr[t] = exp(l10 - l00);
            Qy[t] = exp(l01 - l00);
            Tx[t] = exp((l11 - l01) - (l10 - l00));
        }
        const int chunk_rows = kLabBuf / rx.len;
        for (int r = rbeg; r < rend; r++) {
            const int y = ry.start + r;
            if ((r - rbeg) % chunk_rows == 0) {
                // the labels of the next rows of this wave, loaded in one go
                const int nr = rend - r < chunk_rows ? rend - r : chunk_rows;
                for (int t = lane; t < nr * rx.len; t += 64)
                    labs[wv][t] = a.labels[((int64_t)n * a.H + y + t / rx.len) * a.W + rx.start + t % rx.len];
                __builtin_amdgcn_wave_barrier();
            }
            const uint8_t* lab_row = &labs[wv][((r - rbeg) % chunk_rows) * rx.len];
            int e0, e1;
            bool ecl;
            double ly;
            src_coord_hd(y, a.h, a.H, e0, e1, ly, ecl);
            const double wy0 = 1.0 - ly, wy1 = ly;
            if (r > rbeg) {
#pragma unroll
                for (int t = 0; t < KT; t++) {
                    Er[t] *= Qy[t];
                    Rr[t] *= Tx[t];
                }
            }
            double E[KT], alo[KT], ahi[KT], olo[KT], ohi[KT];
#pragma unroll
            for (int t = 0; t < KT; t++) {
                E[t] = Er[t];
                alo[t] = ahi[t] = olo[t] = ohi[t] = 0.0;
            }
            for (int c = 0; c < rx.len; c++) {
                const double lx = wxs[c];
                const double wx0 = 1.0 - lx, wx1 = lx;
                if (c > 0) {
#pragma unroll
                    for (int t = 0; t < KT; t++) E[t] *= Rr[t];
                }
                double s = 0.0;
#pragma unroll
                for (int t = 0; t < KT; t++) s += E[t];
                s = wave_sum_f64(s);
                const double cp = invP / s;
                // softmax part of the gradient: E / s / P
#pragma unroll
                for (int t = 0; t < KT; t++) {
                    const double g = E[t] * cp;
                    alo[t] += wx0 * g;
                    ahi[t] += wx1 * g;
                }
                // one-hot part: the label's lane collects the pixel's column weights
                const int lab = lab_row[c];
                bad |= lab >= K;
                const bool mine = lane == (lab & 63);
#pragma unroll
                for (int t = 0; t < KT; t++)
                    if ((lab >> 6) == t && mine) {
                        olo[t] += wx0;
                        ohi[t] += wx1;
                    }
                // loss: log(s) + m - l(label); the logs are taken 64 pixels at a time,
                // the label logits at the end of the row from the one-hot weights
                luni += m;
                if ((pc & 63) == lane) sv = s;
                pc++;
                if ((pc & 63) == 0) lsum += log(sv);
            }
#pragma unroll
            for (int t = 0; t < KT; t++) {
                const double glo = alo[t] - olo[t] * invP, ghi = ahi[t] - ohi[t] * invP;
                G00[t] += wy0 * glo;
                G01[t] += wy0 * ghi;
                G10[t] += wy1 * glo;
                G11[t] += wy1 * ghi;
                // sum over the row's pixels labelled k of l_k = the corners' bilinear mix
                llab += (wy0 * (c00[t] * olo[t] + c01[t] * ohi[t]) + wy1 * (c10[t] * olo[t] + c11[t] * ohi[t])) *
                        scale;
            }
        }
    }
    if (lane < (pc & 63)) lsum += log(sv);
    lsum = wave_sum_f64(lsum - llab);
#pragma unroll
    for (int t = 0; t < KT; t++) {
        const int k = lane + 64 * t;
        if (k < K) {
            double* o = red + (int64_t)wv * 4 * K;
            o[k] = G00[t];
            o[K + k] = G01[t];
            o[2 * K + k] = G10[t];
            o[3 * K + k] = G11[t];
        }
    }
    if (lane == 0) {
        wl[wv] = lsum + luni;
        if (bad) set_status(a.status, ISEG_DEV_RANGE);
    }
    __syncthreads();
    const int64_t cid = ((int64_t)n * a.nry + sy) * a.nrx + sx;
    double* out = a.cell + cid * 4 * K;
    for (int t = threadIdx.x; t < 4 * K; t += blockDim.x)
        out[t] = ((red[t] + red[4 * K + t]) + red[8 * K + t]) + red[12 * K + t];
    if (threadIdx.x == 0) a.cell_loss[cid] = ((wl[0] + wl[1]) + wl[2]) + wl[3];
}

// grad[n,i,j,k]: sum over the cells with a corner at (i, j), in cell order
// (row runs, then column runs, then corners); one block per (n, i)
__global__ __launch_bounds__(256) void k_ce_combine(const CeCellArgs a)
{
    const int n = blockIdx.y, i = blockIdx.x;
    __shared__ int ys_lo, ys_hi;
    __shared__ int2 xs[256];             // column run range per low-res column
    if (threadIdx.x == 0) {
        int lo = a.nry, hi = -1;
        for (int s = 0; s < a.nry; s++)
            if (a.ry[s].i0 == i || a.ry[s].i1 == i) {
                lo = s < lo ? s : lo;
                hi = s;
            }
        ys_lo = lo;
        ys_hi = hi;
    }
    for (int j = threadIdx.x; j < a.w; j += blockDim.x) {
        int lo = a.nrx, hi = -1;
        for (int s = 0; s < a.nrx; s++)
            if (a.rx[s].i0 == j || a.rx[s].i1 == j) {
                lo = s < lo ? s : lo;
                hi = s;
            }
        xs[j] = make_int2(lo, hi);
    }
    __syncthreads();
    const int wk = a.w * a.K;
    uint64_t mx = 0;
    for (int e = threadIdx.x; e < wk; e += blockDim.x) {
        const int j = e / a.K, k = e % a.K;
        double acc = 0.0;
        for (int s = ys_lo; s <= ys_hi; s++) {
            const Run ry = a.ry[s];
            for (int g = xs[j].x; g <= xs[j].y; g++) {
                const Run rx = a.rx[g];
                const double* c = a.cell + (((int64_t)n * a.nry + s) * a.nrx + g) * 4 * a.K + k;
                if (ry.i0 == i && rx.i0 == j) acc += c[0];
                if (ry.i0 == i && rx.i1 == j) acc += c[a.K];
                if (ry.i1 == i && rx.i0 == j) acc += c[2 * a.K];
                if (ry.i1 == i && rx.i1 == j) acc += c[3 * a.K];
            }
        }
        a.grad[((int64_t)n * a.h + i) * wk + e] = acc;
        const uint64_t b = (uint64_t)__double_as_longlong(acc) & 0x7fffffffffffffffull;
        mx = b > mx ? b : mx;
    }
    block_store_max_u64(mx, a.part);
}

// smallest e with |v| < 2^e for the positive double with bits mb (frexp's exponent)
__device__ __forceinline__ int frexp_exp_bits64(uint64_t mb)
{
    const int E = (int)(mb >> 52);
    const uint64_t man = mb & 0xfffffffffffffull;
    if (E == 0) return bitlen_u64(man) - 1074;
    return E - 1022;
}

__global__ __launch_bounds__(256) void k_ce_quant(const CeCellArgs a, int64_t nparts, int bits,
                                                  int8_t* __restrict__ err, int32_t* err_exp, double* loss)
{
    const uint64_t mb = reduce_partials_u64(a.part, nparts);
    const int64_t total = (int64_t)a.N * a.h * a.w * a.K;
    const bool range_ok = logit_exp_ok(*a.logit_exp);
    if (!range_ok || mb >= 0x7ff0000000000000ull) {
        // logits outside the region's domain, or a NaN / infinite gradient:
        // flag it, zero codes, NaN loss
        if (blockIdx.x == 0 && threadIdx.x == 0) {
            set_status(a.status, range_ok ? ISEG_DEV_NONFINITE : ISEG_DEV_RANGE);
            *err_exp = 1 - bits;
            if (loss) *loss = __longlong_as_double(0x7ff8000000000000ll);
        }
        for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
             e += (int64_t)gridDim.x * blockDim.x)
            err[e] = 0;
        return;
    }
    const int b = mb ? frexp_exp_bits64(mb) : 0;
    if (blockIdx.x == 0) {
        if (threadIdx.x == 0) *err_exp = b + 1 - bits;
        // mean loss: cell losses summed in a fixed tree order
        __shared__ double red[256];
        double s = 0.0;
        const int64_t cells = (int64_t)a.N * a.nry * a.nrx;
        for (int64_t r = threadIdx.x; r < cells; r += blockDim.x) s += a.cell_loss[r];
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
int launch_cells(const CeCellArgs& a, size_t lds, hipStream_t s)
{
    if (!lds_limit((const void*)k_ce_cells<KT>, lds))
        return ISEG_ERR_DEVICE;
    hipLaunchKernelGGL(k_ce_cells<KT>, dim3((unsigned)a.nrx, (unsigned)a.nry, (unsigned)a.N), dim3(256), lds, s, a);
    return launch_ok();
}

}  // namespace

// workspace: [max][cells][cell losses][grad (if not given)][max partials]
static size_t ce_cell_bytes(int64_t N, int64_t nry, int64_t nrx, int64_t K)
{
    return align256((size_t)(N * nry * nrx * 4 * K) * 8);
}

extern "C" size_t iseg_softmax_ce_ws(int64_t N, int64_t h, int64_t w, int64_t K, int64_t H, int64_t W)
{
    if (N < 1 || h < 1 || w < 1 || K < 1 || H < h || W < w || h > 64 || w > 64 || H > 32767 || W > 32767)
        return 0;
    Run tmp[kMaxRuns];
    const int nry = make_runs((int)h, (int)H, tmp), nrx = make_runs((int)w, (int)W, tmp);
    if (nry < 0 || nrx < 0) return 0;
    return 256 + ce_cell_bytes(N, nry, nrx, K) +
           align256((size_t)(N * nry * nrx) * 8) + align256((size_t)(N * h * w * K) * 8) +
           align256((size_t)(N * h) * 8);
}

extern "C" int iseg_softmax_ce(const int8_t* logits, const int32_t* logit_exp, const uint8_t* labels, int64_t N,
                               int64_t h, int64_t w, int64_t K, int64_t H, int64_t W, int32_t bits, double* loss,
                               double* grad, int8_t* err, int32_t* err_exp, void* ws, size_t ws_bytes,
                               int32_t* dev_status, hipStream_t stream)
{
    if (N < 1 || h < 1 || w < 1 || K < 1 || H < h || W < w || bits < 2 || bits > 8) return ISEG_ERR_ARG;
    if (!logits || !logit_exp || !labels || !err || !err_exp) return ISEG_ERR_ARG;
    if (K > 256 || h > 64 || w > 64 || H > 32767 || W > 32767 || N > 65535) return ISEG_ERR_UNSUPPORTED;
    const size_t need = iseg_softmax_ce_ws(N, h, w, K, H, W);
    if (need == 0) return ISEG_ERR_UNSUPPORTED;
    if (!ws || ws_bytes < need) return ISEG_ERR_WORKSPACE;
    CeCellArgs a{};
    a.logits = logits; a.logit_exp = logit_exp; a.labels = labels;
    a.N = (int32_t)N; a.h = (int32_t)h; a.w = (int32_t)w; a.K = (int32_t)K; a.H = (int32_t)H; a.W = (int32_t)W;
    a.nry = make_runs((int)h, (int)H, a.ry);
    a.nrx = make_runs((int)w, (int)W, a.rx);
    for (int i = 0; i < a.nrx; i++)
        if (a.rx[i].len > kMaxRunLen) return ISEG_ERR_UNSUPPORTED;
    a.status = dev_status;
    char* p = (char*)ws;
    p += 256;
    a.cell = (double*)p;
    p += ce_cell_bytes(N, a.nry, a.nrx, K);
    a.cell_loss = (double*)p;
    p += align256((size_t)(N * a.nry * a.nrx) * 8);
    double* gws = (double*)p;
    p += align256((size_t)(N * h * w * K) * 8);
    a.part = (uint64_t*)p;
    a.grad = grad ? grad : gws;
    int rc;
    const size_t lds = (size_t)((4 * K + 15) & ~(int64_t)15) + (size_t)(kCellWaves * 4 * K) * 8;
    const int kt = (int)((K + 63) / 64);
    rc = kt == 1 ? launch_cells<1>(a, lds, stream)
       : kt == 2 ? launch_cells<2>(a, lds, stream)
       : kt == 3 ? launch_cells<3>(a, lds, stream)
                 : launch_cells<4>(a, lds, stream);
    if (rc) return rc;
    hipLaunchKernelGGL(k_ce_combine, dim3((unsigned)h, (unsigned)N), dim3(256), 0, stream, a);
    if ((rc = launch_ok())) return rc;
    const int64_t nlow = N * h * w * K;
    hipLaunchKernelGGL(k_ce_quant, dim3(grid_for(nlow, 256, 2048)), dim3(256), 0, stream, a, N * h, (int)bits, err,
                       err_exp, loss);
    return launch_ok();
}

// ---------------------------------------------------------------------------
// MSE loss against one-hot labels (the FCN8s loss): L = mean over the N H W K
// elements of (y - t)^2, t = [k == label], and E1 = SQ(2 (y - t) / (N H W K))
// (Eq. 4 / 16) decided exactly.  With g = min(y_exp, 0), every y - t is an
// integer V on the grid 2^g: V = c 2^(y_exp - g) - t 2^-g.  The gradient is
// V 2^(g+1) / D (D = N H W K), its scale 2^u the smallest power of two above
// max|V| 2^(g+1) / D, and a code floor(V 2^(k-1-ce) / D + 1/2) with ce the
// smallest e with max|V| < D 2^e (u = ce + g + 1).  The loss is summed per
// block in float64 and the partials in a fixed order.
// ---------------------------------------------------------------------------
namespace {
struct MseArgs {
    const int8_t* y;
    const int32_t* y_exp;
    const uint8_t* labels;
    int64_t n;               // N H W K
    int32_t K;
    uint64_t* pmax;          // [gridDim.x] max |V|
    double* psum;            // [gridDim.x] sum V^2
    int32_t* status;
};

__device__ __forceinline__ int64_t mse_v(const MseArgs& a, int64_t i, int g, int ye)
{
    const int64_t pix = i / a.K;
    const int k = (int)(i - pix * a.K);
    const int lab = a.labels[pix];
    const int64_t t = lab == k ? 1 : 0;
    return (int64_t)a.y[i] * ((int64_t)1 << (ye - g)) - t * ((int64_t)1 << (-g));
}

__device__ __forceinline__ bool mse_exp_ok(int32_t e) { return e >= -60 && e <= 40; }

__global__ __launch_bounds__(256) void k_mse_part(MseArgs a)
{
    __shared__ double sd[256];
    const int32_t ye = *a.y_exp;
    const bool ok = mse_exp_ok(ye);
    if (!ok && blockIdx.x == 0 && threadIdx.x == 0) set_status(a.status, ISEG_DEV_RANGE);
    const int g = ye < 0 ? ye : 0;
    uint64_t m = 0;
    double s = 0.0;
    bool bad = false;
    if (ok)
        for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < a.n;
             i += (int64_t)gridDim.x * blockDim.x) {
            bad |= a.labels[i / a.K] >= a.K;
            const int64_t v = mse_v(a, i, g, ye);
            const uint64_t av = (uint64_t)(v < 0 ? -v : v);
            m = av > m ? av : m;
            s += (double)v * (double)v;
        }
    if (bad) set_status(a.status, ISEG_DEV_RANGE);
    block_store_max_u64(m, a.pmax);
    sd[threadIdx.x] = s;
    __syncthreads();
    for (int o = 128; o > 0; o >>= 1) {
        if ((int)threadIdx.x < o) sd[threadIdx.x] += sd[threadIdx.x + o];
        __syncthreads();
    }
    if (threadIdx.x == 0) a.psum[blockIdx.x] = sd[0];
}

__global__ __launch_bounds__(256) void k_mse_codes(MseArgs a, int nparts, int bits, int8_t* __restrict__ err,
                                                   int32_t* err_exp, double* loss)
{
    const int32_t ye = *a.y_exp;
    const bool ok = mse_exp_ok(ye);
    const int g = ye < 0 ? ye : 0;
    const uint64_t M = reduce_partials_u64(a.pmax, nparts);
    const i128 D = (i128)a.n;
    const int ce = M ? ceil_pow2_exp128((i128)M, D) : 0;
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        if (M) {
            *err_exp = ce + g + 2 - bits;
        } else {
            int lg = 0;                              // ceil(log2 D)
            while (((int64_t)1 << lg) < a.n) lg++;
            *err_exp = g + 1 - lg;
        }
        double s = 0.0;
        for (int b = 0; b < nparts; b++) s += a.psum[b];
        if (loss) *loss = ok ? ldexp(s, 2 * g) / (double)a.n : __longlong_as_double(0x7ff8000000000000ll);
    }
    const int sh = bits - 1 - ce;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < a.n;
         i += (int64_t)gridDim.x * blockDim.x) {
        int8_t code = 0;
        if (ok && M) code = (int8_t)clamp_k128(rhu128((i128)mse_v(a, i, g, ye), sh, D), bits);
        err[i] = code;
    }
}
}  // namespace

extern "C" size_t iseg_mse_onehot_ws(int64_t n) { return n > 0 ? 256 + 2 * align256(2048 * 8) : 0; }

extern "C" int iseg_mse_onehot(const int8_t* y, const int32_t* y_exp, const uint8_t* labels, int64_t N, int64_t H,
                               int64_t W, int64_t K, int32_t bits, double* loss, int8_t* err, int32_t* err_exp,
                               void* ws, size_t ws_bytes, int32_t* dev_status, hipStream_t stream)
{
    if (N < 1 || H < 1 || W < 1 || K < 1 || bits < 2 || bits > 8) return ISEG_ERR_ARG;
    if (!y || !y_exp || !labels || !err || !err_exp) return ISEG_ERR_ARG;
    if (K > 256 || N * H * W * K > ((int64_t)1 << 40)) return ISEG_ERR_UNSUPPORTED;
    const int64_t n = N * H * W * K;
    if (!ws || ws_bytes < iseg_mse_onehot_ws(n)) return ISEG_ERR_WORKSPACE;
    MseArgs a{};
    a.y = y; a.y_exp = y_exp; a.labels = labels; a.n = n; a.K = (int32_t)K; a.status = dev_status;
    a.pmax = (uint64_t*)((char*)ws + 256);
    a.psum = (double*)((char*)ws + 256 + align256(2048 * 8));
    const unsigned grid = grid_for(n, 256 * 8, 2048);
    hipLaunchKernelGGL(k_mse_part, dim3(grid), dim3(256), 0, stream, a);
    int rc = launch_ok();
    if (rc) return rc;
    hipLaunchKernelGGL(k_mse_codes, dim3(grid_for(n, 256 * 4, 4096)), dim3(256), 0, stream, a, (int)grid,
                       (int)bits, err, err_exp, loss);
    return launch_ok();
}
