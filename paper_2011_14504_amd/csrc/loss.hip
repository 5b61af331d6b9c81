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
    int16_t ylo[64], yhi[64];  // per low-res row: first and last row run touching it
    int16_t xlo[64], xhi[64];  // per low-res column: likewise for column runs
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

// One block per cell (three per CU: occupancy hides the latency of each
// cell's loads and barriers).  A wave takes P = 64 / L rows of the cell at a time, one
// row per group of L lanes; lane l of a group holds the classes l + L t
// (t < KT).  Along a row the exps follow the cell's multiplicative recurrence
// (one multiply per pixel and class), the softmax denominator is a group-wide
// sum (DPP steps within a row of 16 lanes, no readlane) and one reciprocal per
// pixel scales the gradient; two pixels of a row are in flight per step.  The
// cell's per-class constants (the exp at its first pixel, the x- and y-step
// ratios, the change of the x-step per row) are computed once per block; a
// row's starting values are integer powers of them.  The one-hot part of the
// gradient collects in LDS (one region per wave and group, added to by the
// lane that owns the pixel's label with no-return LDS atomics, so no wait),
// the corner sums of the groups are added in group order, then those of the
// waves in wave order.
constexpr int kCellWaves = 4;
constexpr int kMaxRunLen = 256;
constexpr int kLabPre = 4;        // label bytes per lane loaded ahead (a pass of up to 256 pixels)

// v + v[lane ^ O] (O = 16, 32) by gfx950's cross-row swaps; the pair comes
// back in a lane-dependent order, and the sum is the same bits either way
template <int O>
__device__ __forceinline__ double swap_sum_f64(double v)
{
    const uint64_t b = (uint64_t)__double_as_longlong(v);
    const uint32_t lo = (uint32_t)b, hi = (uint32_t)(b >> 32);
    uint32_t l0, l1, h0, h1;
    if constexpr (O == 16) {
        const auto rl = __builtin_amdgcn_permlane16_swap(lo, lo, false, false);
        const auto rh = __builtin_amdgcn_permlane16_swap(hi, hi, false, false);
        l0 = rl[0]; l1 = rl[1]; h0 = rh[0]; h1 = rh[1];
    } else {
        const auto rl = __builtin_amdgcn_permlane32_swap(lo, lo, false, false);
        const auto rh = __builtin_amdgcn_permlane32_swap(hi, hi, false, false);
        l0 = rl[0]; l1 = rl[1]; h0 = rh[0]; h1 = rh[1];
    }
    const double x = __longlong_as_double((long long)(((uint64_t)h0 << 32) | l0));
    const double y = __longlong_as_double((long long)(((uint64_t)h1 << 32) | l1));
    return x + y;
}

template <int O>
__device__ __forceinline__ double swap_max_f64(double v)
{
    const uint64_t b = (uint64_t)__double_as_longlong(v);
    const uint32_t lo = (uint32_t)b, hi = (uint32_t)(b >> 32);
    uint32_t l1, h1;
    if constexpr (O == 16) {
        const auto rl = __builtin_amdgcn_permlane16_swap(lo, lo, false, false);
        const auto rh = __builtin_amdgcn_permlane16_swap(hi, hi, false, false);
        l1 = rl[0] == lo && rh[0] == hi ? rl[1] : rl[0];
        h1 = rl[0] == lo && rh[0] == hi ? rh[1] : rh[0];
    } else {
        const auto rl = __builtin_amdgcn_permlane32_swap(lo, lo, false, false);
        const auto rh = __builtin_amdgcn_permlane32_swap(hi, hi, false, false);
        l1 = rl[0] == lo && rh[0] == hi ? rl[1] : rl[0];
        h1 = rl[0] == lo && rh[0] == hi ? rh[1] : rh[0];
    }
    return fmax(v, __longlong_as_double((long long)(((uint64_t)h1 << 32) | l1)));
}

// group-wide (L = 16: one DPP row, L = 32: two) sum / max of a double, by
// steps whose partner pairs are symmetric: every lane of the group ends with
// the same bits
template <int L>
__device__ __forceinline__ double group_sum_f64(double v)
{
    v += dpp_f64<0xB1>(v);
    v += dpp_f64<0x4E>(v);
    v += dpp_f64<0x141>(v);
    v += dpp_f64<0x140>(v);
    if constexpr (L == 32) v = swap_sum_f64<16>(v);
    return v;
}

template <int L>
__device__ __forceinline__ double group_max_f64(double v)
{
    v = fmax(v, dpp_f64<0xB1>(v));
    v = fmax(v, dpp_f64<0x4E>(v));
    v = fmax(v, dpp_f64<0x141>(v));
    v = fmax(v, dpp_f64<0x140>(v));
    if constexpr (L == 32) v = swap_max_f64<16>(v);
    return v;
}

// sum of a value over the P groups of a wave (lanes l, l + L, ...), the same
// bits in every lane: pairs of groups first, then pairs of pairs
template <int L>
__device__ __forceinline__ double groups_sum_f64(double v)
{
    if constexpr (L == 16) v = swap_sum_f64<16>(v);
    return swap_sum_f64<32>(v);
}

// b^e, e >= 0, by squaring
__device__ __forceinline__ double pow_int(double b, int e)
{
    double r = 1.0;
    while (e) {
        if (e & 1) r *= b;
        b *= b;
        e >>= 1;
    }
    return r;
}

// pairwise sum of KT values
template <int KT>
__device__ __forceinline__ double tree_sum(const double* v)
{
    double t[KT];
#pragma unroll
    for (int i = 0; i < KT; i++) t[i] = v[i];
#pragma unroll
    for (int w = 1; w < KT; w *= 2)
#pragma unroll
        for (int i = 0; i + w < KT; i += 2 * w) t[i] += t[i + w];
    return t[0];
}

// a / s for s > 0 (a normal double, here at least exp(-256)): hardware
// reciprocal, two Newton steps and one correction of the quotient
__device__ __forceinline__ double div_pos(double a, double s)
{
    double r = __builtin_amdgcn_rcp(s);
    r = fma(fma(-s, r, 1.0), r, r);
    r = fma(fma(-s, r, 1.0), r, r);
    const double q = a * r;
    return fma(fma(-s, q, a), r, q);
}

__device__ __forceinline__ void lds_add_f64(double* p, double v)
{
    (void)__hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

template <int L, int KT>
__global__ __launch_bounds__(256, 3) void k_ce_cells(const CeCellArgs a)
{
    constexpr int P = 64 / L;
    static_assert(L == 16 || L == 32, "group width");
    extern __shared__ __align__(16) char smem[];
    __shared__ double wxs[kMaxRunLen];                     // column weight lambda_x per pixel of the run
    __shared__ double wl[kCellWaves];
    __shared__ uint8_t labs[kCellWaves][P][kMaxRunLen];    // labels of the rows a wave has in flight
    const int n = blockIdx.z, sy = blockIdx.y, sx = blockIdx.x;
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int grp = lane / L, lig = lane % L;
    const int K = a.K, wk = a.w * a.K;
    const Run ry = a.ry[sy], rx = a.rx[sx];
    const int j0 = rx.i0, j1 = rx.i1, len = rx.len;
    // LDS: the four corner columns of both source rows [4][K] (codes), the
    // per-class constants [4][K], and per wave P one-hot regions [2][K]
    // (reused for the wave's corner sums [4][K] at the end)
    int8_t* C0 = (int8_t*)smem;
    double* cst = (double*)(smem + ((4 * K + 15) & ~15));
    double* oh = cst + 4 * K;
    // labels of a pass (rows base .. base + P - 1 of the run): up to kLabPre
    // bytes per lane through registers, so a pass's loads can be issued early
    const uint8_t* lab_base = a.labels + ((int64_t)n * a.H + ry.start) * a.W + rx.start;
    auto lab_load = [&](int base, uint32_t* v) {
#pragma unroll
        for (int q = 0; q < kLabPre; q++) {
            const int t = lane + 64 * q, rr = base + t / len;
            v[q] = t < P * len && rr < ry.len ? lab_base[(int64_t)rr * a.W + t % len] : 0u;
        }
    };
    auto lab_store = [&](int base, const uint32_t* v) {
#pragma unroll
        for (int q = 0; q < kLabPre; q++) {
            const int t = lane + 64 * q;
            if (t < P * len) labs[wv][t / len][t % len] = (uint8_t)v[q];
        }
        for (int t = lane + 64 * kLabPre; t < P * len; t += 64) {
            const int rr = base + t / len;
            labs[wv][t / len][t % len] = rr < ry.len ? lab_base[(int64_t)rr * a.W + t % len] : (uint8_t)0;
        }
    };
    uint32_t lpre[kLabPre];
    lab_load(wv * P, lpre);
    const int8_t* r0 = a.logits + ((int64_t)n * a.h + ry.i0) * wk;
    const int8_t* r1 = a.logits + ((int64_t)n * a.h + ry.i1) * wk;
    for (int t = threadIdx.x; t < K; t += blockDim.x) {
        C0[t] = r0[j0 * K + t];
        C0[K + t] = r0[j1 * K + t];
        C0[2 * K + t] = r1[j0 * K + t];
        C0[3 * K + t] = r1[j1 * K + t];
    }
    for (int c = threadIdx.x; c < len; c += blockDim.x) {
        int e0, e1;
        bool ecl;
        double lx;
        src_coord_hd(rx.start + c, a.w, a.W, e0, e1, lx, ecl);
        wxs[c] = lx;
    }
    for (int t = threadIdx.x; t < kCellWaves * P * 2 * K; t += blockDim.x) oh[t] = 0.0;
    __syncthreads();
    // outside the documented range the outputs are discarded (k_ce_quant)
    const double scale = logit_exp_ok(*a.logit_exp) ? ldexp(1.0, *a.logit_exp) : 0.0;
    const double invP = 1.0 / ((double)a.N * (double)a.H * (double)a.W);

    // the cell's max logit (each group covers every class: the same m everywhere)
    double m = -INFINITY;
#pragma unroll
    for (int t = 0; t < KT; t++) {
        const int k = lig + L * t;
        if (k < K) m = fmax(m, fmax(fmax((double)C0[k], (double)C0[K + k]),
                                    fmax((double)C0[2 * K + k], (double)C0[3 * K + k])) * scale);
    }
    m = group_max_f64<L>(m);

    // per class: exp at the first pixel, x-step and y-step ratios, and the
    // factor by which the x-step changes from row to row
    {
        int d0, d1;
        bool dcl;
        double ly0, ly1;
        src_coord_hd(ry.start, a.h, a.H, d0, d1, ly0, dcl);
        src_coord_hd(ry.start + (ry.len > 1 ? 1 : 0), a.h, a.H, d0, d1, ly1, dcl);
        const double lx0 = wxs[0], lx1 = wxs[len > 1 ? 1 : 0];
        for (int k = threadIdx.x; k < K; k += blockDim.x) {
            const double c00 = C0[k], c01 = C0[K + k], c10 = C0[2 * K + k], c11 = C0[3 * K + k];
            const double l00 = interp(c00, c01, c10, c11, 1.0 - lx0, lx0, 1.0 - ly0, ly0, scale);
            const double l10 = interp(c00, c01, c10, c11, 1.0 - lx1, lx1, 1.0 - ly0, ly0, scale);
            const double l01 = interp(c00, c01, c10, c11, 1.0 - lx0, lx0, 1.0 - ly1, ly1, scale);
            const double l11 = interp(c00, c01, c10, c11, 1.0 - lx1, lx1, 1.0 - ly1, ly1, scale);
            cst[k] = exp(l00 - m);
            cst[K + k] = exp(l10 - l00);
            cst[2 * K + k] = exp(l01 - l00);
            cst[3 * K + k] = exp((l11 - l01) - (l10 - l00));
        }
    }
    lab_store(wv * P, lpre);
    __syncthreads();

    double G00[KT], G01[KT], G10[KT], G11[KT];
#pragma unroll
    for (int t = 0; t < KT; t++) G00[t] = G01[t] = G10[t] = G11[t] = 0.0;
    double lsum = 0.0, llab = 0.0, sv = 1.0;
    int pc = 0;
    bool bad = false;
    double* ohg = oh + (int64_t)((wv * P + grp) * 2) * K;
    const uint8_t* lab_row = labs[wv][grp];
    for (int base = wv * P; base < ry.len; base += kCellWaves * P) {
        const int row = base + grp;
        const bool live = row < ry.len;
        const bool more = base + kCellWaves * P < ry.len;
        if (more) lab_load(base + kCellWaves * P, lpre);     // the next pass's labels, in flight meanwhile
        int e0, e1;
        bool ecl;
        double ly;
        src_coord_hd(ry.start + (live ? row : 0), a.h, a.H, e0, e1, ly, ecl);
        const double wy0 = 1.0 - ly, wy1 = ly;
        double E[KT], R[KT], alo[KT], ahi[KT];
#pragma unroll
        for (int t = 0; t < KT; t++) {
            const int k = lig + L * t;
            const bool on = k < K;
            E[t] = on && live ? cst[k] * pow_int(cst[2 * K + k], row) : 0.0;
            R[t] = on ? cst[K + k] * pow_int(cst[3 * K + k], live ? row : 0) : 1.0;
            alo[t] = ahi[t] = 0.0;
        }
        // one pixel of the row: softmax part of the gradient E / s / P folded
        // into the row's two columns; one-hot part by the label's lane; the
        // loss log(s) + m - l(label), logs taken L pixels at a time and the
        // label logits at the end of the row from the one-hot weights
        auto pixel = [&](const double* Ev, double s, double lx, int lab, bool on) {
            const double cp = on ? div_pos(invP, s) : 0.0;
            const double c0 = (1.0 - lx) * cp, c1 = lx * cp;
#pragma unroll
            for (int t = 0; t < KT; t++) {
                alo[t] = fma(c0, Ev[t], alo[t]);
                ahi[t] = fma(c1, Ev[t], ahi[t]);
            }
            if (on) {
                bad |= lab >= K;
                if (lab < K && lig == lab % L) {
                    lds_add_f64(&ohg[lab], 1.0 - lx);
                    lds_add_f64(&ohg[K + lab], lx);
                }
                if ((pc % L) == lig) sv = s;
                pc++;
                if (pc % L == 0) lsum += log(sv);
            }
        };
        for (int c = 0; c < len; c += 2) {
            const bool two = c + 1 < len;
            const double lxa = wxs[c], lxb = wxs[two ? c + 1 : c];
            const int laba = lab_row[c], labb = lab_row[two ? c + 1 : c];
            double E1[KT];
#pragma unroll
            for (int t = 0; t < KT; t++) E1[t] = E[t] * R[t];
            const double sa = group_sum_f64<L>(tree_sum<KT>(E));
            const double sb = group_sum_f64<L>(tree_sum<KT>(E1));
            pixel(E, sa, lxa, laba, live);
            pixel(E1, sb, lxb, labb, live && two);
#pragma unroll
            for (int t = 0; t < KT; t++) E[t] = E1[t] * R[t];
        }
        if (live) {
#pragma unroll
            for (int t = 0; t < KT; t++) {
                const int k = lig + L * t;
                if (k < K) {
                    const double olo = ohg[k], ohi = ohg[K + k];
                    ohg[k] = 0.0;
                    ohg[K + k] = 0.0;
                    const double glo = alo[t] - olo * invP, ghi = ahi[t] - ohi * invP;
                    G00[t] += wy0 * glo;
                    G01[t] += wy0 * ghi;
                    G10[t] += wy1 * glo;
                    G11[t] += wy1 * ghi;
                    // sum over the row's pixels labelled k of l_k = the corners' bilinear mix
                    llab += (wy0 * ((double)C0[k] * olo + (double)C0[K + k] * ohi) +
                             wy1 * ((double)C0[2 * K + k] * olo + (double)C0[3 * K + k] * ohi)) * scale;
                }
            }
        }
        __builtin_amdgcn_wave_barrier();
        if (more) lab_store(base + kCellWaves * P, lpre);
        __builtin_amdgcn_wave_barrier();
    }
    if (lig < (pc % L)) lsum += log(sv);
    lsum = wave_sum_f64(lsum - llab);
    const bool anybad = __any(bad);
    // the groups' corner sums, then this wave's into its own LDS region
    double* red = oh + (int64_t)wv * P * 2 * K;             // [4][K], within the wave's one-hot regions
#pragma unroll
    for (int t = 0; t < KT; t++) {
        const double g00 = groups_sum_f64<L>(G00[t]), g01 = groups_sum_f64<L>(G01[t]);
        const double g10 = groups_sum_f64<L>(G10[t]), g11 = groups_sum_f64<L>(G11[t]);
        const int k = lig + L * t;
        if (grp == 0 && k < K) {
            red[k] = g00;
            red[K + k] = g01;
            red[2 * K + k] = g10;
            red[3 * K + k] = g11;
        }
    }
    if (lane == 0) {
        wl[wv] = lsum;
        if (anybad) set_status(a.status, ISEG_DEV_RANGE);
    }
    __syncthreads();
    const int64_t cid = ((int64_t)n * a.nry + sy) * a.nrx + sx;
    double* out = a.cell + cid * 4 * K;
    const int64_t ws = (int64_t)P * 2 * K;
    for (int t = threadIdx.x; t < 4 * K; t += blockDim.x)
        out[t] = ((oh[t] + oh[ws + t]) + oh[2 * ws + t]) + oh[3 * ws + t];
    if (threadIdx.x == 0)
        a.cell_loss[cid] = (((wl[0] + wl[1]) + wl[2]) + wl[3]) + m * ((double)ry.len * (double)len);
}

// grad[n,i,j,k]: sum over the cells with a corner at (i, j), in cell order
// (row runs, then column runs, then corners); one thread per element, a block
// per 256 elements of one low-res row, the runs touching i and j from tables
__global__ __launch_bounds__(256) void k_ce_combine(const CeCellArgs a)
{
    const int n = blockIdx.z, i = blockIdx.y;
    const int wk = a.w * a.K;
    const int e = blockIdx.x * 256 + threadIdx.x;
    uint64_t mx = 0;
    if (e < wk) {
        const int j = e / a.K, k = e - j * a.K;
        double acc = 0.0;
        for (int s = a.ylo[i]; s <= a.yhi[i]; s++) {
            const Run ry = a.ry[s];
            for (int g = a.xlo[j]; g <= a.xhi[j]; g++) {
                const Run rx = a.rx[g];
                const double* c = a.cell + (((int64_t)n * a.nry + s) * a.nrx + g) * 4 * a.K + k;
                if (ry.i0 == i && rx.i0 == j) acc += c[0];
                if (ry.i0 == i && rx.i1 == j) acc += c[a.K];
                if (ry.i1 == i && rx.i0 == j) acc += c[2 * a.K];
                if (ry.i1 == i && rx.i1 == j) acc += c[3 * a.K];
            }
        }
        a.grad[((int64_t)n * a.h + i) * wk + e] = acc;
        mx = (uint64_t)__double_as_longlong(acc) & 0x7fffffffffffffffull;
    }
    mx = block_max_u64(mx);
    if (threadIdx.x == 0) a.part[((int64_t)n * a.h + i) * gridDim.x + blockIdx.x] = mx;
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

template <int L, int KT>
int launch_cells(const CeCellArgs& a, hipStream_t s)
{
    const size_t lds = (size_t)((4 * a.K + 15) & ~15) + (size_t)(4 * a.K) * 8 +
                       (size_t)(kCellWaves * (64 / L) * 2 * a.K) * 8;
    if (!lds_limit((const void*)k_ce_cells<L, KT>, lds))
        return ISEG_ERR_DEVICE;
    hipLaunchKernelGGL((k_ce_cells<L, KT>), dim3((unsigned)a.nrx, (unsigned)a.nry, (unsigned)a.N), dim3(256), lds,
                       s, a);
    return launch_ok();
}

// first and last run touching each low-res index (an empty range: lo > hi)
void run_ranges(const Run* runs, int nr, int n_low, int16_t* lo, int16_t* hi)
{
    for (int i = 0; i < n_low; i++) {
        lo[i] = (int16_t)nr;
        hi[i] = -1;
        for (int s = 0; s < nr; s++)
            if (runs[s].i0 == i || runs[s].i1 == i) {
                if (s < lo[i]) lo[i] = (int16_t)s;
                hi[i] = (int16_t)s;
            }
    }
}

// max |grad| partials: one per combine block
int64_t ce_nparts(int64_t N, int64_t h, int64_t w, int64_t K) { return N * h * ceil_div64(w * K, 256); }

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
           align256((size_t)ce_nparts(N, h, w, K) * 8);
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
    run_ranges(a.ry, a.nry, (int)h, a.ylo, a.yhi);
    run_ranges(a.rx, a.nrx, (int)w, a.xlo, a.xhi);
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
    // groups of 16 lanes up to 128 classes (KT rounded up to an instantiated
    // width), else 32: more classes per lane cost occupancy
    const int kt16 = (int)((K + 15) / 16), kt32 = (int)((K + 31) / 32);
    rc = kt16 <= 1   ? launch_cells<16, 1>(a, stream)
       : kt16 <= 2   ? launch_cells<16, 2>(a, stream)
       : kt16 <= 4   ? launch_cells<16, 4>(a, stream)
       : kt16 <= 6   ? launch_cells<16, 6>(a, stream)
       : kt16 <= 8   ? launch_cells<16, 8>(a, stream)
       : kt32 <= 5   ? launch_cells<32, 5>(a, stream)
       : kt32 <= 6   ? launch_cells<32, 6>(a, stream)
                     : launch_cells<32, 8>(a, stream);
    if (rc) return rc;
    const unsigned cx = (unsigned)ceil_div64(w * K, 256);
    hipLaunchKernelGGL(k_ce_combine, dim3(cx, (unsigned)h, (unsigned)N), dim3(256), 0, stream, a);
    if ((rc = launch_ok())) return rc;
    const int64_t nlow = N * h * w * K;
    hipLaunchKernelGGL(k_ce_quant, dim3(grid_for(nlow, 256 * 4, 512)), dim3(256), 0, stream, a,
                       ce_nparts(N, h, w, K), (int)bits, err, err_exp, loss);
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
