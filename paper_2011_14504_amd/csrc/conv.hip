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

// a convolution is timed as a whole entry-point call (ProfScope), not per kernel
#undef ISEG_TIMED_LAUNCH
#define ISEG_TIMED_LAUNCH(kid, stream, ...) \
    do {                                    \
        (void)(kid);                        \
        hipLaunchKernelGGL(__VA_ARGS__);    \
    } while (0)

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
    int16_t* out16;               // staged [Mrows][Nout] (int16 path)
    uint8_t* tshift;              // per (row tile, column tile) staging shift
    uint64_t* pmax;               // per-block max |sum| partials (may be null)
    int8_t* out8;                 // final SQ codes (second pass of the two-pass path)
    const int32_t* exp_a;         // operand exponents and the result exponent (second pass)
    const int32_t* exp_b;
    int32_t* out_exp;
    int64_t npmax;                // partials written by the first pass
    int64_t Mrows;
    int32_t Nout, Kred, Ci;
    int32_t Hs, Ws, Ho, Wo;
    int32_t R, S;
    int32_t sh, sw, ph, pw, dh, dw;
    int32_t tap_balance;          // every tile skips a tap: split its live steps evenly
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

template <int MODE>
int launch_igemm_generic(const IgemmArgs& a, hipStream_t s, int64_t* nblk);

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
    if (a.pmax) block_store_max_u64(mx, a.pmax);
}

// Implicit GEMM for Ci % 64 == 0: the k-loop runs tap-major in 64-channel
// chunks, so each step is one tap and one contiguous channel chunk.  Source
// offsets of a thread's rows are recomputed only when the tap changes; LDS
// is double-buffered (one barrier per step) and the next step's global
// loads are in flight while the current step's MFMAs run.
template <int MODE, int BM, int BN>
__global__ __launch_bounds__(256) void k_conv_igemm_tap(IgemmArgs a)
{
    constexpr int PA = BM * 4 / 256;
    constexpr int PB = BN * 4 / 256;
    constexpr int WM = BM / 2, WN = BN / 2;
    constexpr int TM = WM / 16, TN = WN / 16;
    __shared__ __attribute__((aligned(16))) int8_t As[2][BM * ROW];
    __shared__ __attribute__((aligned(16))) int8_t Bs[2][BN * ROW];

    const int tid = threadIdx.x;
    const int part = tid & 3;
    const int64_t m0 = (int64_t)blockIdx.x * BM;
    const int n0 = blockIdx.y * BN;
    const int nchunk = a.Ci / BK;
    const int nk = a.R * a.S * nchunk;

    RowPix rp[PA];
#pragma unroll
    for (int j = 0; j < PA; j++) rp[j] = row_pix(a, m0 + ((tid >> 2) + 64 * j));
    const int8_t* brow[PB];
#pragma unroll
    for (int j = 0; j < PB; j++) {
        int n = n0 + (tid >> 2) + 64 * j;
        brow[j] = n < a.Nout ? a.wmat + (int64_t)n * a.Kred + part * 16 : nullptr;
    }

    int64_t soff[PA];
    auto set_tap = [&](int tap) {
        int r = tap / a.S, s = tap - (tap / a.S) * a.S;
#pragma unroll
        for (int j = 0; j < PA; j++) {
            int64_t sp = src_pixel<MODE>(a, rp[j], r, s);
            soff[j] = sp < 0 ? -1 : sp * a.Ci + part * 16;
        }
    };
    int4 ra[PA], rb[PB];
    auto load = [&](int kb, int cc) {
#pragma unroll
        for (int j = 0; j < PA; j++)
            ra[j] = soff[j] >= 0 ? *(const int4*)(a.src + soff[j] + cc * BK) : make_int4(0, 0, 0, 0);
#pragma unroll
        for (int j = 0; j < PB; j++)
            rb[j] = brow[j] ? *(const int4*)(brow[j] + (int64_t)kb * BK) : make_int4(0, 0, 0, 0);
    };
    auto store = [&](int buf) {
#pragma unroll
        for (int j = 0; j < PA; j++) *(int4*)&As[buf][((tid >> 2) + 64 * j) * ROW + part * 16] = ra[j];
#pragma unroll
        for (int j = 0; j < PB; j++) *(int4*)&Bs[buf][((tid >> 2) + 64 * j) * ROW + part * 16] = rb[j];
    };

    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int lrow = lane & 15, lk = (lane >> 4) * 16;
    v4i acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; i++)
#pragma unroll
        for (int j = 0; j < TN; j++) acc[i][j] = (v4i){0, 0, 0, 0};

    int tap = 0, cc = 0;
    set_tap(0);
    load(0, 0);
    store(0);
    __syncthreads();
    for (int kb = 0; kb < nk; kb++) {
        const bool more = kb + 1 < nk;
        if (more) {
            if (++cc == nchunk) { cc = 0; set_tap(++tap); }
            load(kb + 1, cc);
        }
        const int8_t* A = As[kb & 1];
        const int8_t* B = Bs[kb & 1];
        v4i fa[TM], fb[TN];
#pragma unroll
        for (int i = 0; i < TM; i++) fa[i] = *(const v4i*)&A[(wm * WM + i * 16 + lrow) * ROW + lk];
#pragma unroll
        for (int j = 0; j < TN; j++) fb[j] = *(const v4i*)&B[(wn * WN + j * 16 + lrow) * ROW + lk];
#pragma unroll
        for (int i = 0; i < TM; i++)
#pragma unroll
            for (int j = 0; j < TN; j++)
                acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[i], fb[j], acc[i][j], 0, 0, 0);
        if (more) store((kb + 1) & 1);
        __syncthreads();
    }

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
    if (a.pmax) block_store_max_u64(mx, a.pmax);
}

// ---------------------------------------------------------------------------
// Implicit GEMM with direct-to-LDS loads (Ci % 64 == 0, Nout % BN == 0).
//
// Each step (one tap, one 64-channel chunk) stages a 128 x 64-byte A tile and
// a BN x 64-byte B tile with global_load_lds_dwordx4: a wave's instruction
// writes 64 lanes x 16 bytes contiguously, i.e. 16 tile rows.  Pieces are
// placed with an XOR swizzle (16-byte slot = part ^ ((row >> 1) & 3)) instead
// of row padding: for the fragment reads of v_mfma_i32_16x16x64_i8 (lane l
// reads row l % 16, slot l / 16) this is the placement that gfx950's LDS
// serves without bank conflicts (measured with SQ_LDS_BANK_CONFLICT; the
// (row >> 2) and padded-row placements both conflict).  Taps falling into
// padding load from a zero page.
// kStages LDS buffers keep kStages - 1 steps of loads in flight; vmcnt tracks
// the DMA completions and one barrier per step publishes a stage.
// ---------------------------------------------------------------------------
__device__ __attribute__((aligned(64))) int8_t g_conv_zero[64];
#ifndef ISEG_IGEMM_STAGES
#define ISEG_IGEMM_STAGES 3      // LDS stages of the direct-to-LDS implicit GEMM
#endif
constexpr int kStages = ISEG_IGEMM_STAGES;
#ifndef ISEG_IGEMM_TAPSKIP
#define ISEG_IGEMM_TAPSKIP 1     // skip the taps that read only padding for a whole tile (stride 1)
#endif

// Taps of a stride-1 conv that read only padding for every row of the tile
// [m0, m0 + rows): the source pixel is the output pixel shifted by a per-tap
// constant (r dh - ph forward; ph - r dh for backward-data), so a tap is
// empty when the tile's output-row or output-column range, shifted, misses
// the source extent.  A tile crossing an image (row) keeps the full row
// (column) range.  Returns the mask of taps to run.
template <int MODE>
__host__ __device__ __forceinline__ uint64_t live_taps(const IgemmArgs& a, int64_t m0, int rows)
{
    const int RS = a.R * a.S;                 // <= 64 (igemm_dma_ok)
    const uint64_t all = RS == 64 ? ~0ull : (1ull << RS) - 1;
    if (!ISEG_IGEMM_TAPSKIP || RS == 1 || a.sh != 1 || a.sw != 1) return all;
    const int64_t m1 = m0 + rows - 1;
    const int64_t hw = (int64_t)a.Ho * a.Wo;
    const int64_t n0 = m0 / hw, n1 = m1 / hw;
    const int32_t p0 = (int32_t)(m0 - n0 * hw), p1 = (int32_t)(m1 - n1 * hw);
    int oh_lo = p0 / a.Wo, oh_hi = p1 / a.Wo;
    int ow_lo = p0 - oh_lo * a.Wo, ow_hi = p1 - oh_hi * a.Wo;
    if (n0 != n1) { oh_lo = 0; oh_hi = a.Ho - 1; }
    if (n0 != n1 || oh_lo != oh_hi) { ow_lo = 0; ow_hi = a.Wo - 1; }
    uint64_t mask = 0;
    for (int r = 0; r < a.R; r++) {
        const int cr = MODE == MODE_FWD ? r * a.dh - a.ph : a.ph - r * a.dh;
        if (oh_hi + cr < 0 || oh_lo + cr >= a.Hs) continue;
        for (int t = 0; t < a.S; t++) {
            const int cs = MODE == MODE_FWD ? t * a.dw - a.pw : a.pw - t * a.dw;
            if (ow_hi + cs < 0 || ow_lo + cs >= a.Ws) continue;
            mask |= 1ull << (r * a.S + t);
        }
    }
    return mask;
}

typedef __attribute__((address_space(3))) void lds_void_t;

__device__ __forceinline__ void dma16(const void* g, int8_t* lds_wave_base)
{
    __builtin_amdgcn_global_load_lds(g, (lds_void_t*)lds_wave_base, 16, 0, 0);
}

// wait until at most n vector-memory operations of this wave are outstanding
template <int N>
__device__ __forceinline__ void wait_vm()
{
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

__device__ __forceinline__ int swz(int row, int part) { return row * 64 + ((part ^ ((row >> 1) & 3)) << 4); }

// row -> (image, output row, output column) in 32-bit arithmetic (Mrows < 2^31)
__device__ __forceinline__ RowPix row_pix32(const IgemmArgs& a, int64_t m)
{
    RowPix rp;
    rp.ok = m < a.Mrows;
    const uint32_t mm = rp.ok ? (uint32_t)m : 0u;
    const uint32_t hw = (uint32_t)a.Ho * (uint32_t)a.Wo;
    rp.n = (int32_t)(mm / hw);
    const uint32_t rem = mm - (uint32_t)rp.n * hw;
    rp.oh = (int32_t)(rem / (uint32_t)a.Wo);
    rp.ow = (int32_t)(rem - (uint32_t)rp.oh * (uint32_t)a.Wo);
    return rp;
}

// epilogues: raw int32 sums; int16 staging; tile max only (first pass of the
// two-pass path); final SQ codes from the global max (second pass); int32
// partial sums of one split of the reduction
enum { EPI_RAW = 0, EPI_STAGE16 = 1, EPI_MAX = 2, EPI_Q8 = 3, EPI_PART = 4 };

// wait until this wave's LDS reads have returned and at most n vector-memory
// operations are outstanding
template <int N>
__device__ __forceinline__ void wait_vm_lgkm0()
{
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (0 << 8));
}

// Staging of the exact int32 sums as int16 with a per-tile right shift
// t = max(0, bitlen(tile max) - 15): floor(acc / 2^t) fits int16, and since
// the tensor's requant shift r = bitlen(max) - 7 is >= t + 1 whenever t > 0,
// rounding floor(acc / 2^t) half-up by the remaining r - t bits gives the same
// code as rounding acc by r (2^(r-1) is a multiple of 2^t, so the dropped low
// bits can never carry into the rounding position).
//
// Pipeline: step kb's A/B fragments are read from LDS into registers one step
// ahead, so the ds_reads of step kb + 1 run under the MFMAs of step kb; once a
// step's fragments are in registers its LDS stage is free and receives the
// DMA of step kb + kStages, which keeps kStages - 1 steps of loads in flight.
template <int MODE, int BM, int BN, int EPI, bool PIPE>
__global__ __launch_bounds__(256) void k_conv_igemm_dma(IgemmArgs a)
{
    constexpr int WM = BM / 2, WN = BN / 2;  // 2 x 2 waves
    constexpr int TM = WM / 16, TN = WN / 16;
    constexpr int NA = BM / 64;              // A instructions per wave and step (16 rows each)
    constexpr int NB = BN / 64;              // B instructions per wave and step
    constexpr int LPW = NA + NB;             // DMA loads per wave and step
    constexpr int SA = BM * 64, SB = BN * 64;
    extern __shared__ __attribute__((aligned(16))) int8_t smem[];   // [kStages][SA + SB]

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    // XCD-aware tile order: consecutive pixel tiles go to one XCD (blocks are
    // dealt to the 8 XCDs round-robin), so halo rows are shared in its L2
    const int nbx = gridDim.x;
    int bx = blockIdx.x;
    if ((nbx & 7) == 0) bx = (bx & 7) * (nbx >> 3) + (bx >> 3);
    const int64_t m0 = (int64_t)bx * BM;
    const int n0 = blockIdx.y * BN;
    const int nchunk = a.Ci / BK;
    // the taps this tile runs (all but those reading only padding).  Steps
    // are (tap, chunk) pairs, tap-major; a split (blockIdx.z of gridDim.z)
    // owns the same step range [kb0, kb1) in every tile, so the blocks of one
    // split read one slice of W (shared in L2), and runs the live steps in it.
    const int RS = a.R * a.S;
    const int64_t vr = a.Mrows - m0;
    const uint64_t tmask = live_taps<MODE>(a, m0, vr < BM ? (int)vr : BM);
    // When every tile skips a tap (tap_balance, decided on the host) the live
    // steps themselves are split evenly: the splits of one tile then stay
    // balanced, at the cost of W slices that differ between tiles.
    const int nk_full = a.tap_balance ? __builtin_popcountll(tmask) * nchunk : RS * nchunk;
    const int kb0 = (int)((int64_t)nk_full * blockIdx.z / gridDim.z);
    const int kb1 = (int)((int64_t)nk_full * (blockIdx.z + 1) / gridDim.z);
    int nk = 0;
    if (a.tap_balance) {
        nk = kb1 - kb0;
    } else {
        for (int t = 0; t < RS; t++) {
            if (!((tmask >> t) & 1)) continue;
            const int lo = kb0 > t * nchunk ? kb0 : t * nchunk;
            const int hi = kb1 < (t + 1) * nchunk ? kb1 : (t + 1) * nchunk;
            nk += hi > lo ? hi - lo : 0;
        }
    }

    // this lane's DMA pieces: row (16 * instr + lane / 4) in slot lane % 4
    const int rin = lane >> 2;
    const int part = (lane & 3) ^ ((rin >> 1) & 3);
    RowPix rp[NA];
#pragma unroll
    for (int j = 0; j < NA; j++) rp[j] = row_pix32(a, m0 + 16 * (wave + 4 * j) + rin);
    const int8_t* brow[NB];
#pragma unroll
    for (int j = 0; j < NB; j++) brow[j] = a.wmat + (int64_t)(n0 + 16 * (wave + 4 * j) + rin) * a.Kred + part * 16;

    int64_t soff[NA];
    auto set_tap = [&](int tap) {
        const int r = tap / a.S, s = tap - (tap / a.S) * a.S;
#pragma unroll
        for (int j = 0; j < NA; j++) {
            const int64_t sp = src_pixel<MODE>(a, rp[j], r, s);
            soff[j] = sp < 0 ? -1 : sp * a.Ci + part * 16;
        }
    };
    // (tap, chunk) of the step being issued: balanced, the (kb0 / nchunk)-th
    // live tap; aligned, the first live step at or after kb0
    int ltap = kb0 / nchunk, lcc = kb0 - (kb0 / nchunk) * nchunk;
    if (a.tap_balance) {
        uint64_t mm = tmask;
        for (int i = kb0 / nchunk; i > 0 && mm; i--) mm &= mm - 1;
        ltap = mm ? __builtin_ctzll(mm) : RS;
    } else if (ltap < RS && !((tmask >> ltap) & 1)) {
        const uint64_t rest = ltap + 1 < 64 ? tmask >> (ltap + 1) : 0ull;
        ltap = rest ? ltap + 1 + __builtin_ctzll(rest) : RS;
        lcc = 0;
    }
    auto issue = [&](int kb) {               // kb: step within this split
        int8_t* st = smem + (kb % kStages) * (SA + SB);
#pragma unroll
        for (int j = 0; j < NA; j++) {
            const void* g = soff[j] >= 0 ? (const void*)(a.src + soff[j] + lcc * BK) : (const void*)g_conv_zero;
            dma16(g, st + (wave + 4 * j) * 1024);
        }
        const int64_t boff = (int64_t)ltap * a.Ci + lcc * BK;
#pragma unroll
        for (int j = 0; j < NB; j++) dma16(brow[j] + boff, st + SA + (wave + 4 * j) * 1024);
        if (++lcc == nchunk) {
            lcc = 0;
            const uint64_t rest = ltap + 1 < 64 ? tmask >> (ltap + 1) : 0ull;
            ltap = rest ? ltap + 1 + __builtin_ctzll(rest) : RS;
            if (ltap < RS) set_tap(ltap);
        }
    };

    const int wm = wave >> 1, wn = wave & 1;
    const int lrow = lane & 15, lpart = lane >> 4;
    v4i acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; i++)
#pragma unroll
        for (int j = 0; j < TN; j++) acc[i][j] = (v4i){0, 0, 0, 0};

    auto frags = [&](int kb, v4i* fa, v4i* fb) {
        const int8_t* A = smem + (kb % kStages) * (SA + SB);
        const int8_t* B = A + SA;
#pragma unroll
        for (int i = 0; i < TM; i++) fa[i] = *(const v4i*)&A[swz(wm * WM + i * 16 + lrow, lpart)];
#pragma unroll
        for (int j = 0; j < TN; j++) fb[j] = *(const v4i*)&B[swz(wn * WN + j * 16 + lrow, lpart)];
        // keep the reads ahead of the MFMAs that follow (they run under them)
        __builtin_amdgcn_sched_barrier(0);
    };
    auto mma = [&](const v4i* fa, const v4i* fb) {
#pragma unroll
        for (int i = 0; i < TM; i++)
#pragma unroll
            for (int j = 0; j < TN; j++)
                acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[i], fb[j], acc[i][j], 0, 0, 0);
    };
    // Every step slot issues LPW loads per wave (past the last step: loads of
    // the zero page into the stage just freed), so the number of loads in
    // flight behind any step is the same in every trip and one wait count fits.
    auto issue_any = [&](int kb) {
        if (kb < nk) {
            issue(kb);
        } else {
            int8_t* st = smem + (kb % kStages) * (SA + SB);
#pragma unroll
            for (int j = 0; j < LPW; j++) dma16(g_conv_zero, st + (wave + 4 * j) * 1024);
        }
    };
    // make step kb + 1 visible to every wave and free step kb's stage for the
    // DMA of step kb + kStages (steps kb + 2 .. kb + kStages - 1 stay in flight)
    static_assert(kStages >= 2 && (kStages - 1) * LPW < 64, "vmcnt range");
    auto advance = [&](int kb) {
        wait_vm_lgkm0<(kStages - 2) * LPW>();
        // a plain barrier: __syncthreads() would also drain every DMA in flight
        __builtin_amdgcn_s_barrier();
        issue_any(kb + kStages);
    };

    if (nk > 0) set_tap(ltap);
#pragma unroll
    for (int p = 0; p < kStages; p++) issue_any(p);
    uint64_t gmax = 0;
    if (EPI == EPI_Q8) gmax = reduce_partials_u64(a.pmax, a.npmax);
    wait_vm<(kStages - 1) * LPW>();           // step 0 has landed
    __builtin_amdgcn_s_barrier();
    if (PIPE) {
        // fragments one step ahead in registers: the ds_reads of step kb + 1
        // are issued before the MFMAs of step kb
        v4i fa[TM], fb[TN], na[TM], nb[TN];
        if (nk > 0) frags(0, fa, fb);
        for (int kb = 0; kb < nk; kb++) {
            const bool more = kb + 1 < nk;
            if (more) {
                advance(kb);
                frags(kb + 1, na, nb);
            }
            mma(fa, fb);
            if (more) {
#pragma unroll
                for (int i = 0; i < TM; i++) fa[i] = na[i];
#pragma unroll
                for (int j = 0; j < TN; j++) fb[j] = nb[j];
            }
        }
    } else {
        // one fragment set: the other resident wave of the SIMD covers the
        // LDS latency
        v4i fa[TM], fb[TN];
        for (int kb = 0; kb < nk; kb++) {
            frags(kb, fa, fb);
            mma(fa, fb);
            if (kb + 1 < nk) advance(kb);
        }
    }
    wait_vm<0>();                             // the zero-page loads still in flight

    // rows of this block that exist (the last row tile may be ragged)
    const int vrows = a.Mrows - m0 < BM ? (int)(a.Mrows - m0) : BM;
    if (EPI == EPI_PART) {
        int32_t* out = a.out + (int64_t)blockIdx.z * a.Mrows * a.Nout;
#pragma unroll
        for (int i = 0; i < TM; i++)
#pragma unroll
            for (int j = 0; j < TN; j++) {
                const int n = n0 + wn * WN + j * 16 + lrow;
#pragma unroll
                for (int e = 0; e < 4; e++) {
                    const int row = wm * WM + i * 16 + lpart * 4 + e;
                    if (row < vrows) out[(m0 + row) * a.Nout + n] = acc[i][j][e];
                }
            }
        return;
    }
    if (EPI == EPI_RAW) {
        uint32_t mx = 0;
#pragma unroll
        for (int i = 0; i < TM; i++)
#pragma unroll
            for (int j = 0; j < TN; j++) {
                const int n = n0 + wn * WN + j * 16 + lrow;
#pragma unroll
                for (int e = 0; e < 4; e++) {
                    const int row = wm * WM + i * 16 + lpart * 4 + e;
                    if (row < vrows) {
                        const int32_t v = acc[i][j][e];
                        a.out[(m0 + row) * a.Nout + n] = v;
                        const uint32_t av = (uint32_t)(v < 0 ? -v : v);
                        mx = av > mx ? av : mx;
                    }
                }
            }
        if (a.pmax) block_store_max_u64(mx, a.pmax);
        return;
    }
    uint32_t mx = 0;
#pragma unroll
    for (int i = 0; i < TM; i++)
#pragma unroll
        for (int j = 0; j < TN; j++)
#pragma unroll
            for (int e = 0; e < 4; e++) {
                const int row = wm * WM + i * 16 + lpart * 4 + e;
                const int32_t v = acc[i][j][e];
                const uint32_t av = row < vrows ? (uint32_t)(v < 0 ? -v : v) : 0u;
                mx = av > mx ? av : mx;
            }
    if (EPI == EPI_MAX) {
        block_store_max_u64(mx, a.pmax);
        return;
    }
    if (EPI == EPI_Q8) {
        // final SQ codes with r = bitlen(global max) - 7, staged through LDS
        const int rq = gmax ? (64 - __builtin_clzll(gmax)) - 7 : 0;
        if (blockIdx.x == 0 && blockIdx.y == 0 && tid == 0) *a.out_exp = *a.exp_a + *a.exp_b + rq;
        const int rs = rq > 0 ? rq - 1 : 0, ls = rq > 0 ? 0 : -rq;
        constexpr int RB8 = BN + 16;          // codes per LDS row (16-byte pad: bank spread)
        __syncthreads();                      // every wave is done with the stage buffers
#pragma unroll
        for (int i = 0; i < TM; i++)
#pragma unroll
            for (int j = 0; j < TN; j++)
#pragma unroll
                for (int e = 0; e < 4; e++) {
                    const int row = wm * WM + i * 16 + lpart * 4 + e;
                    const int32_t x = acc[i][j][e];
                    int32_t c = rq > 0 ? ((x >> rs) + 1) >> 1 : x << ls;
                    c = c > 127 ? 127 : (c < -127 ? -127 : c);
                    smem[row * RB8 + wn * WN + j * 16 + lrow] = (int8_t)c;
                }
        __syncthreads();
        constexpr int CPR = BN / 16;          // 16-byte chunks per row
#pragma unroll
        for (int k = 0; k < BM * CPR / 256; k++) {
            const int c = tid + k * 256;
            const int row = c / CPR, cc = c - (c / CPR) * CPR;
            if (row < vrows)
                *(int4*)(a.out8 + (m0 + row) * a.Nout + n0 + cc * 16) = *(const int4*)&smem[row * RB8 + cc * 16];
        }
        return;
    }
    // int16 staging: tile max -> shift, shifted tile through LDS, 16-byte stores
    __shared__ uint32_t wmax[4];
    mx = wave_max_u32(mx);
    if (lane == 0) wmax[wave] = mx;
    __syncthreads();                          // also: every wave is done with the stage buffers
    uint32_t tmax = wmax[0];
#pragma unroll
    for (int w = 1; w < 4; w++) tmax = wmax[w] > tmax ? wmax[w] : tmax;
    const int t = tmax ? max(0, 32 - __builtin_clz(tmax) - 15) : 0;
    constexpr int RS16 = BN + 8;              // int16 per LDS row (16-byte pad: bank spread)
    int16_t* T = (int16_t*)smem;
#pragma unroll
    for (int i = 0; i < TM; i++)
#pragma unroll
        for (int j = 0; j < TN; j++)
#pragma unroll
            for (int e = 0; e < 4; e++) {
                const int row = wm * WM + i * 16 + lpart * 4 + e;
                T[row * RS16 + wn * WN + j * 16 + lrow] = (int16_t)(acc[i][j][e] >> t);
            }
    __syncthreads();
    constexpr int CPR = BN / 8;               // 16-byte chunks per row
#pragma unroll
    for (int k = 0; k < BM * CPR / 256; k++) {
        const int c = tid + k * 256;
        const int row = c / CPR, cc = c - (c / CPR) * CPR;
        if (row < vrows)
            *(int4*)(a.out16 + (m0 + row) * a.Nout + n0 + cc * 8) = *(const int4*)&T[row * RS16 + cc * 8];
    }
    if (tid == 0) {
        a.tshift[(int64_t)bx * gridDim.y + blockIdx.y] = (uint8_t)t;
        if (a.pmax) a.pmax[(int64_t)blockIdx.y * gridDim.x + blockIdx.x] = tmax;
    }
}

// ---------------------------------------------------------------------------
// Short reductions with final codes (Kred <= 256: at most four 64-byte steps),
// persistent over row tiles.  A block owns one BN-column slice of W, staged in
// LDS once for all its tiles, and `tpb` consecutive 128-row tiles.  A tiles
// are double-buffered whole: the loads of tile t + 1 are issued as tile t
// starts, so they run under tile t's MFMAs and epilogue.  The only vector-
// memory operations issued after them are tile t's epilogue stores (SX per
// thread), so "tile t + 1 has landed" is the constant wait vmcnt <= SX; plain
// barriers (no __syncthreads, which would drain the loads in flight) order
// the LDS buffers.  EPI_MAX folds every tile into one running max and leaves
// one partial per block; EPI_Q8 writes the codes from the global max.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void wait_lgkm0()
{
    __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4) | (0 << 8));   // lgkmcnt(0), vmcnt untouched
}

template <int BN, int EPI>
constexpr size_t short_lds_bytes(int nk)
{
    return (size_t)nk * BN * 64 + 2 * (size_t)nk * 128 * 64 + (EPI == EPI_Q8 ? (size_t)128 * (BN + 16) : 0);
}

template <int MODE, int BN, int EPI>
__global__ __launch_bounds__(256) void k_conv_short(IgemmArgs a, int tpb)
{
    constexpr int BM = 128, WM = BM / 2, WN = BN / 2;
    constexpr int TM = WM / 16, TN = WN / 16;
    constexpr int NA = BM / 64, NB = BN / 64;
    constexpr int SA = BM * 64, SB = BN * 64;
    constexpr int RB8 = BN + 16;                          // codes per staging row (16-byte pad)
    constexpr int SX = EPI == EPI_Q8 ? BM * (BN / 16) / 256 : 0;
    static_assert(SX < 64, "vmcnt range");
    extern __shared__ __attribute__((aligned(16))) int8_t smem[];
    const int nk = a.Kred / BK;
    // the staging rows first, at a fixed offset: provably apart from every
    // DMA target, so reading them waits for no load in flight
    constexpr int SE = EPI == EPI_Q8 ? BM * RB8 : 0;
    int8_t* El = smem;                                    // [BM][RB8]
    int8_t* Bl = smem + SE;                               // [nk][SB]
    int8_t* Al = Bl + nk * SB;                            // [2][nk][SA]

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int n0 = blockIdx.y * BN;
    const int64_t nt = (a.Mrows + BM - 1) / BM;
    const int64_t tbeg = (int64_t)blockIdx.x * tpb;
    const int ntile = (int)(nt - tbeg < tpb ? nt - tbeg : tpb);
    const int nchunk = a.Ci / BK;
    const int rin = lane >> 2;
    const int part = (lane & 3) ^ ((rin >> 1) & 3);

    uint64_t gmax = 0;
    if (EPI == EPI_Q8) gmax = reduce_partials_u64(a.pmax, a.npmax);   // before any load is in flight
    const int rq = gmax ? (64 - __builtin_clzll(gmax)) - 7 : 0;
    if (EPI == EPI_Q8 && blockIdx.x == 0 && blockIdx.y == 0 && tid == 0) *a.out_exp = *a.exp_a + *a.exp_b + rq;

    // the block's slice of W for every step
    for (int kb = 0; kb < nk; kb++)
#pragma unroll
        for (int j = 0; j < NB; j++)
            dma16(a.wmat + (int64_t)(n0 + 16 * (wave + 4 * j) + rin) * a.Kred + kb * BK + part * 16,
                  Bl + kb * SB + (wave + 4 * j) * 1024);
    auto issue_tile = [&](int64_t tile, int buf) {
        RowPix rp[NA];
#pragma unroll
        for (int j = 0; j < NA; j++) rp[j] = row_pix32(a, tile * BM + 16 * (wave + 4 * j) + rin);
        int64_t soff[NA];
        int tap = 0, cc = 0;
        for (int kb = 0; kb < nk; kb++) {
            if (cc == 0) {
                const int r = tap / a.S, s = tap - (tap / a.S) * a.S;
#pragma unroll
                for (int j = 0; j < NA; j++) {
                    const int64_t sp = src_pixel<MODE>(a, rp[j], r, s);
                    soff[j] = sp < 0 ? -1 : sp * a.Ci + part * 16;
                }
            }
#pragma unroll
            for (int j = 0; j < NA; j++) {
                const void* g = soff[j] >= 0 ? (const void*)(a.src + soff[j] + cc * BK) : (const void*)g_conv_zero;
                dma16(g, Al + (buf * nk + kb) * SA + (wave + 4 * j) * 1024);
            }
            if (++cc == nchunk) { cc = 0; ++tap; }
        }
    };
    if (ntile > 0) issue_tile(tbeg, 0);

    const int wm = wave >> 1, wn = wave & 1;
    const int lrow = lane & 15, lpart = lane >> 4;
    const int rs = rq > 0 ? rq - 1 : 0, ls = rq > 0 ? 0 : -rq;
    uint32_t run_max = 0;
    for (int t = 0; t < ntile; t++) {
        const int buf = t & 1;
        if (t == 0) wait_vm<0>();                         // W slice and tile 0
        else wait_vm<SX>();                               // tile t (tile t - 1's stores may still run)
        // every wave's part of tile t is in LDS; every wave is done with the
        // other buffer (tile t - 1) and with the staging rows
        __builtin_amdgcn_s_barrier();
        if (t + 1 < ntile) issue_tile(tbeg + t + 1, buf ^ 1);
        v4i acc[TM][TN];
#pragma unroll
        for (int i = 0; i < TM; i++)
#pragma unroll
            for (int j = 0; j < TN; j++) acc[i][j] = (v4i){0, 0, 0, 0};
        for (int kb = 0; kb < nk; kb++) {
            const int8_t* A = Al + (buf * nk + kb) * SA;
            const int8_t* B = Bl + kb * SB;
            v4i fa[TM], fb[TN];
#pragma unroll
            for (int i = 0; i < TM; i++) fa[i] = *(const v4i*)&A[swz(wm * WM + i * 16 + lrow, lpart)];
#pragma unroll
            for (int j = 0; j < TN; j++) fb[j] = *(const v4i*)&B[swz(wn * WN + j * 16 + lrow, lpart)];
#pragma unroll
            for (int i = 0; i < TM; i++)
#pragma unroll
                for (int j = 0; j < TN; j++)
                    acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[i], fb[j], acc[i][j], 0, 0, 0);
        }
        const int64_t m0 = (tbeg + t) * BM;
        const int vrows = a.Mrows - m0 < BM ? (int)(a.Mrows - m0) : BM;
        if (EPI == EPI_MAX) {
#pragma unroll
            for (int i = 0; i < TM; i++)
#pragma unroll
                for (int j = 0; j < TN; j++)
#pragma unroll
                    for (int e = 0; e < 4; e++) {
                        const int row = wm * WM + i * 16 + lpart * 4 + e;
                        const int32_t v = acc[i][j][e];
                        const uint32_t av = row < vrows ? (uint32_t)(v < 0 ? -v : v) : 0u;
                        run_max = av > run_max ? av : run_max;
                    }
        } else {
#pragma unroll
            for (int i = 0; i < TM; i++)
#pragma unroll
                for (int j = 0; j < TN; j++)
#pragma unroll
                    for (int e = 0; e < 4; e++) {
                        const int row = wm * WM + i * 16 + lpart * 4 + e;
                        const int32_t x = acc[i][j][e];
                        int32_t c = rq > 0 ? ((x >> rs) + 1) >> 1 : x << ls;
                        c = c > 127 ? 127 : (c < -127 ? -127 : c);
                        El[row * RB8 + wn * WN + j * 16 + lrow] = (int8_t)c;
                    }
            wait_lgkm0();
            __builtin_amdgcn_s_barrier();                 // the tile's codes are in LDS
            constexpr int CPR = BN / 16;                  // 16-byte chunks per row
            int4 v[SX > 0 ? SX : 1];
#pragma unroll
            for (int k = 0; k < SX; k++) {
                const int c = tid + k * 256;
                v[k] = *(const int4*)&El[(c / CPR) * RB8 + (c % CPR) * 16];
            }
            // every chunk in registers before the guarded stores (kept from
            // being sunk into them, where each would reuse one register set)
#pragma unroll
            for (int k = 0; k < SX; k++) asm volatile("" : "+v"(v[k].x), "+v"(v[k].y), "+v"(v[k].z), "+v"(v[k].w));
#pragma unroll
            for (int k = 0; k < SX; k++) {
                const int c = tid + k * 256;
                const int row = c / CPR, cc = c % CPR;
                if (row < vrows) *(int4*)(a.out8 + (m0 + row) * a.Nout + n0 + cc * 16) = v[k];
            }
        }
    }
    wait_vm<0>();
    if (EPI == EPI_MAX) block_store_max_u64(run_max, a.pmax);
}

// ---------------------------------------------------------------------------
// Short 1x1 stride-1 convolutions with final codes: a plain GEMM
// out[m][n] = sum_k A[m][k] B[n][k] over contiguous pixels, Kred = 64 NK <=
// 256, entirely in registers.  A wave owns 64 output channels, whose B
// fragments stay in VGPRs, and walks blocks of 16 MT pixels, loading the next
// block's A fragments (16 bytes per lane, 1 KB contiguous per 16 pixels)
// while the current block's MFMAs run.  The product is formed as W x A^T, so
// a lane's four results are four consecutive channels of one pixel: one
// packed dword per 16 x 16 tile.  No LDS and no barriers in the loop:
// occupancy is set by registers alone and many loads stay in flight.
// Waves of a block share their pixel blocks when there are >= 4 channel
// groups (their A loads meet in the CU's L1).  EPI_MAX leaves one max
// partial per block; EPI_Q8 writes the codes from the global max.
// ---------------------------------------------------------------------------
template <int NK, int EPI>
__global__ __launch_bounds__(256) void k_gemm_short(IgemmArgs a)
{
    constexpr int MT = NK <= 2 ? 2 : 1;                   // 16-pixel tiles per block of pixels
    constexpr int PB = 16 * MT;
    const int lane = threadIdx.x & 63;
    const int lr = lane & 15, lk = lane >> 4;
    const int ncg = a.Nout / 64;
    const int64_t gw = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int cg = (int)(gw % ncg);
    const int64_t wstride = (int64_t)gridDim.x * 4 / ncg;    // the grid's waves are a multiple of ncg
    const int64_t npb = (a.Mrows + PB - 1) / PB;

    uint64_t gmax = 0;
    if (EPI == EPI_Q8) gmax = reduce_partials_u64(a.pmax, a.npmax);
    const int rq = gmax ? (64 - __builtin_clzll(gmax)) - 7 : 0;
    const int rs = rq > 0 ? rq - 1 : 0, ls = rq > 0 ? 0 : -rq;
    if (EPI == EPI_Q8 && blockIdx.x == 0 && threadIdx.x == 0) *a.out_exp = *a.exp_a + *a.exp_b + rq;

    v4i fb[4][NK];
#pragma unroll
    for (int j = 0; j < 4; j++)
#pragma unroll
        for (int s = 0; s < NK; s++)
            fb[j][s] = *(const v4i*)(a.wmat + (int64_t)(cg * 64 + j * 16 + lr) * a.Kred + s * 64 + lk * 16);
    auto load_a = [&](int64_t pb, v4i (&fa)[MT][NK]) {
#pragma unroll
        for (int i = 0; i < MT; i++) {
            int64_t m = pb * PB + i * 16 + lr;
            m = m < a.Mrows ? m : a.Mrows - 1;             // rows past the end: loaded, never used
            const int8_t* p = a.src + m * a.Kred + lk * 16;
#pragma unroll
            for (int s = 0; s < NK; s++) fa[i][s] = *(const v4i*)(p + s * 64);
        }
    };
    uint32_t mx = 0;
    // one block of PB pixels from fa: acc[j][i][e] is pixel pb PB + 16 i + lr,
    // channel 64 cg + 16 j + 4 lk + e.  Full blocks store unconditionally, so
    // the compiler can count the stores behind the next block's loads.
    auto block = [&](int64_t pb, const v4i (&fa)[MT][NK], bool ragged) {
        v4i acc[4][MT];
#pragma unroll
        for (int j = 0; j < 4; j++)
#pragma unroll
            for (int i = 0; i < MT; i++) acc[j][i] = (v4i){0, 0, 0, 0};
#pragma unroll
        for (int s = 0; s < NK; s++)
#pragma unroll
            for (int j = 0; j < 4; j++)
#pragma unroll
                for (int i = 0; i < MT; i++)
                    acc[j][i] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fb[j][s], fa[i][s], acc[j][i], 0, 0, 0);
#pragma unroll
        for (int i = 0; i < MT; i++) {
            const int64_t m = pb * PB + i * 16 + lr;
            if (ragged && m >= a.Mrows) continue;
#pragma unroll
            for (int j = 0; j < 4; j++) {
                if (EPI == EPI_MAX) {
#pragma unroll
                    for (int e = 0; e < 4; e++) {
                        const int32_t v = acc[j][i][e];
                        const uint32_t av = (uint32_t)(v < 0 ? -v : v);
                        mx = av > mx ? av : mx;
                    }
                } else {
                    uint32_t packed = 0;
#pragma unroll
                    for (int e = 0; e < 4; e++) {
                        const int32_t x = acc[j][i][e];
                        int32_t c = rq > 0 ? ((x >> rs) + 1) >> 1 : x << ls;
                        c = c > 127 ? 127 : (c < -127 ? -127 : c);
                        packed |= (uint32_t)(uint8_t)(int8_t)c << (8 * e);
                    }
                    *(uint32_t*)(a.out8 + m * a.Nout + cg * 64 + j * 16 + lk * 4) = packed;
                }
            }
        }
    };
    const int64_t nfull = a.Mrows / PB;
    int64_t pb = gw / ncg;
    v4i fa[MT][NK], na[MT][NK];
    if (pb < npb) load_a(pb, fa);
    for (; pb < nfull; pb += wstride) {
        const bool more = pb + wstride < npb;
        if (more) load_a(pb + wstride, na);
        block(pb, fa, false);
        if (more) {
#pragma unroll
            for (int i = 0; i < MT; i++)
#pragma unroll
                for (int s = 0; s < NK; s++) fa[i][s] = na[i][s];
        }
    }
    if (pb < npb) block(pb, fa, true);         // the ragged last block, already in fa
    if (EPI == EPI_MAX) block_store_max_u64(mx, a.pmax);
}

// ---------------------------------------------------------------------------
// 3x3, stride-1 convolution from an LDS halo tile (Ci % 64 == 0, Nout % 64 == 0).
//
// A block owns TH = 4 output rows x TW output columns of one image and 64
// output channels; wave w computes output row w.  Per 64-channel chunk the
// block stages the (TH + 2 dh) x (TW + 2 dw) input halo and the 9 x 64 x 64
// weight slice once (direct-to-LDS loads, XOR-swizzled 16-byte slots: slot =
// part ^ ((index >> 2) & 3), so any 16 consecutive pixels or channels are
// conflict-free for ds_read_b128), then runs all nine taps from LDS: the A
// operand of tap (r, s) is the halo shifted by (r dh, s dw).  Backward-data
// with stride 1 is the same convolution over dy with the flipped, transposed
// filter and padding dil (R - 1) - pad.
// ---------------------------------------------------------------------------
struct HaloArgs {
    const int8_t* src;            // [N][Hs][Ws][Ci]
    const int8_t* wmat;           // [Nout][3][3][Ci]
    int32_t* out;                 // raw sums [N][Ho][Wo][Nout] (when out16 is null)
    int16_t* out16;               // staged sums
    uint8_t* tshift;              // per (tile, 64-channel group) staging shift
    int8_t* out8;                 // final SQ codes (second pass of the two-pass path)
    const int32_t* exp_a;         // operand exponents and the result exponent (second pass)
    const int32_t* exp_b;
    int32_t* out_exp;
    uint64_t* pmax;               // per-block max |sum| partials
    int64_t npmax;
    int32_t N, Hs, Ws, Ci, Ho, Wo, Nout;
    int32_t ph, pw, dh, dw;       // input row of output row y and tap r: y - ph + r dh
    int32_t tiles_y, tiles_x;
};

constexpr int kHaloTH = 4;

size_t halo_lds_bytes(int TW, int dh, int dw)
{
    return (size_t)(kHaloTH + 2 * dh) * (TW + 2 * dw) * 64 + 9 * 64 * 64;
}

template <int TW, int EPI>
__global__ __launch_bounds__(256) void k_conv3x3_halo(HaloArgs a)
{
    constexpr int TH = kHaloTH, TM = TW / 16, TN = 4;
    extern __shared__ __attribute__((aligned(16))) int8_t smem[];
    const int HR = TH + 2 * a.dh, HC = TW + 2 * a.dw;
    const int nhalo = HR * HC * 4;                        // 16-byte pieces
    int8_t* halo = smem;
    int8_t* wts = smem + HR * HC * 64;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int nbx = gridDim.x;
    int bx = blockIdx.x;
    if ((nbx & 7) == 0) bx = (bx & 7) * (nbx >> 3) + (bx >> 3);
    const int tx = bx % a.tiles_x, t2 = bx / a.tiles_x;
    const int ty = t2 % a.tiles_y, n = t2 / a.tiles_y;
    const int oy0 = ty * TH, ox0 = tx * TW, k0 = blockIdx.y * 64;
    const int iy0 = oy0 - a.ph, ix0 = ox0 - a.pw;
    const int lrow = lane & 15, lpart = lane >> 4;

    v4i acc[TM][TN];

    // A-operand LDS addresses of fragment 0 for the nine taps: fragment i adds
    // 16 pixels = 1024 bytes and leaves the swizzle phase unchanged
    int aaddr[9];
#pragma unroll
    for (int r = 0; r < 3; r++)
#pragma unroll
        for (int s2 = 0; s2 < 3; s2++) {
            const int p = (wave + r * a.dh) * HC + lrow + s2 * a.dw;
            aaddr[r * 3 + s2] = p * 64 + ((lpart ^ ((p >> 2) & 3)) << 4);
        }
    int baddr[TN];
#pragma unroll
    for (int j = 0; j < TN; j++) {
        const int kk = 16 * j + lrow;
        baddr[j] = kk * 64 + ((lpart ^ ((kk >> 2) & 3)) << 4);
    }
    // halo pieces of this lane: instruction k = wave + 4 u covers pixels
    // 16 k .. 16 k + 15; pixel (hr, hc) advances by 64 per instruction
    const int p0 = 16 * wave + (lane >> 2);
    const int hr0 = p0 / HC, hc0 = p0 - (p0 / HC) * HC;
    // weight pieces: instruction k = wave + 4 j holds tap j (rows of 16
    // channels kk = 16 (wave) + lane / 4 ... ), same lane slot in every tap
    const int wkk = ((wave * 64 + lane) >> 2) & 63;
    const int wpart = (lane & 3) ^ ((wkk >> 2) & 3);
    const int wtap0 = (wave * 64 + lane) >> 8;
    const int8_t* wsrc = a.wmat + ((int64_t)(k0 + wkk) * 9 + wtap0) * a.Ci + wpart * 16;

    const int nchunk = a.Ci / 64;
    uint64_t gmax = 0;
    for (int cc = 0; cc < nchunk; cc++) {
        if (cc) __syncthreads();                          // the previous chunk's reads are done
        {
            int hr = hr0, hc = hc0;
            for (int k = wave; k * 64 < nhalo; k += 4) {
                const int q = k * 64 + lane;
                if (q < nhalo) {
                    const int p = q >> 2;
                    const int part = (q & 3) ^ ((p >> 2) & 3);
                    const int iy = iy0 + hr, ix = ix0 + hc;
                    const bool v = (unsigned)iy < (unsigned)a.Hs && (unsigned)ix < (unsigned)a.Ws;
                    const void* g = v ? (const void*)(a.src + (((int64_t)n * a.Hs + iy) * a.Ws + ix) * a.Ci +
                                                      cc * 64 + part * 16)
                                      : (const void*)g_conv_zero;
                    dma16(g, halo + k * 1024);
                }
                hc += 64;
                while (hc >= HC) { hc -= HC; ++hr; }
            }
        }
        // instruction wave + 4 j covers pieces (wave + 4 j) * 64 + lane: tap =
        // wtap0 + j (four instructions per tap), same channel row and slot
#pragma unroll
        for (int j = 0; j < 9; j++)
            dma16(wsrc + (int64_t)j * a.Ci + cc * 64, wts + (wave + 4 * j) * 1024);
        // second pass: the global max, read while the first chunk is in flight
        if (EPI == EPI_Q8 && cc == 0) gmax = reduce_partials_u64(a.pmax, a.npmax);
        wait_vm<0>();
        __syncthreads();
#pragma unroll
        for (int t = 0; t < 9; t++) {
            v4i fa[TM], fb[TN];
#pragma unroll
            for (int i = 0; i < TM; i++) fa[i] = *(const v4i*)&halo[aaddr[t] + 1024 * i];
#pragma unroll
            for (int j = 0; j < TN; j++) fb[j] = *(const v4i*)&wts[t * 4096 + baddr[j]];
            if (t == 0 && cc == 0) {              // first product: no accumulator to clear
#pragma unroll
                for (int i = 0; i < TM; i++)
#pragma unroll
                    for (int j = 0; j < TN; j++)
                        acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[i], fb[j], (v4i){0, 0, 0, 0}, 0, 0, 0);
            } else {
#pragma unroll
                for (int i = 0; i < TM; i++)
#pragma unroll
                    for (int j = 0; j < TN; j++)
                        acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[i], fb[j], acc[i][j], 0, 0, 0);
            }
        }
    }

    // acc[i][j][e]: output (row wave, column 16 i + 4 lpart + e), channel k0 + 16 j + lrow
    const int oy = oy0 + wave;
    const int64_t rowbase = ((int64_t)n * a.Ho + oy) * a.Wo;
    if (EPI == EPI_RAW) {
        if (oy < a.Ho) {
#pragma unroll
            for (int i = 0; i < TM; i++)
#pragma unroll
                for (int e = 0; e < 4; e++) {
                    const int ox = ox0 + 16 * i + 4 * lpart + e;
                    if (ox < a.Wo) {
#pragma unroll
                        for (int j = 0; j < TN; j++)
                            a.out[(rowbase + ox) * a.Nout + k0 + 16 * j + lrow] = acc[i][j][e];
                    }
                }
        }
        return;
    }
    const int vcols = a.Wo - ox0 < TW ? a.Wo - ox0 : TW;
    if (EPI == EPI_Q8) {
        // codes = SQ(acc) with r = bitlen(global max) - 7; rhu(acc, r) = ((acc >> (r - 1)) + 1) >> 1
        const uint64_t M = gmax;
        const int r = M ? (64 - __builtin_clzll(M)) - 7 : 0;
        if (blockIdx.x == 0 && blockIdx.y == 0 && tid == 0) *a.out_exp = *a.exp_a + *a.exp_b + r;
        constexpr int RB8 = 64 + 16;                  // bytes per LDS row of the code tile
        int8_t* T = smem + (wave * TW + 4 * lpart) * RB8 + lrow;
        __syncthreads();                              // every wave is done with the halo
        const int rs = r > 0 ? r - 1 : 0, ls = r > 0 ? 0 : -r;
#pragma unroll
        for (int i = 0; i < TM; i++)
#pragma unroll
            for (int e = 0; e < 4; e++)
#pragma unroll
                for (int j = 0; j < TN; j++) {
                    const int32_t v = acc[i][j][e];
                    int32_t c = r > 0 ? ((v >> rs) + 1) >> 1 : v << ls;
                    c = c > 127 ? 127 : (c < -127 ? -127 : c);
                    T[(16 * i + e) * RB8 + 16 * j] = (int8_t)c;
                }
        __syncthreads();
        if (oy < a.Ho) {
            // wave w stores tile row w: chunk (pixel lane / 4 + 16 u, channels 16 (lane % 4) ..)
            const int8_t* T0 = smem + (wave * TW + (lane >> 2)) * RB8 + (lane & 3) * 16;
            int8_t* g = a.out8 + ((rowbase + ox0 + (lane >> 2)) * a.Nout + k0 + (lane & 3) * 16);
#pragma unroll
            for (int u = 0; u < TW / 16; u++)
                if ((lane >> 2) + 16 * u < vcols)
                    *(int4*)(g + (int64_t)16 * u * a.Nout) = *(const int4*)&T0[16 * u * RB8];
        }
        return;
    }
    __shared__ uint32_t wmax[4];
    // tile max |acc| via running max and min (max3/min3 take two values per op)
    int32_t vmax = 0, vmin = 0;
    if (oy < a.Ho) {
        if (vcols == TW) {
#pragma unroll
            for (int i = 0; i < TM; i++)
#pragma unroll
                for (int e = 0; e < 4; e++)
#pragma unroll
                    for (int j = 0; j < TN; j += 2) {
                        vmax = max(vmax, max(acc[i][j][e], acc[i][j + 1][e]));
                        vmin = min(vmin, min(acc[i][j][e], acc[i][j + 1][e]));
                    }
        } else {
#pragma unroll
            for (int i = 0; i < TM; i++)
#pragma unroll
                for (int e = 0; e < 4; e++)
                    if (16 * i + 4 * lpart + e < vcols) {
#pragma unroll
                        for (int j = 0; j < TN; j += 2) {
                            vmax = max(vmax, max(acc[i][j][e], acc[i][j + 1][e]));
                            vmin = min(vmin, min(acc[i][j][e], acc[i][j + 1][e]));
                        }
                    }
        }
    }
    uint32_t mx = (uint32_t)max(vmax, -vmin);
    mx = wave_max_u32(mx);
    if (EPI == EPI_MAX) {
        const uint64_t bm = block_max_u64(mx);
        if (tid == 0) a.pmax[(int64_t)blockIdx.y * gridDim.x + blockIdx.x] = bm;
        return;
    }
    if (lane == 0) wmax[wave] = mx;
    __syncthreads();                                      // also: all waves are done with the halo
    uint32_t tmax = wmax[0];
#pragma unroll
    for (int w = 1; w < 4; w++) tmax = wmax[w] > tmax ? wmax[w] : tmax;
    const int tsh = tmax ? max(0, 32 - __builtin_clz(tmax) - 15) : 0;
    constexpr int RS16 = 64 + 8;
    int16_t* T = (int16_t*)smem + (wave * TW + 4 * lpart) * RS16 + lrow;
#pragma unroll
    for (int i = 0; i < TM; i++)
#pragma unroll
        for (int e = 0; e < 4; e++)
#pragma unroll
            for (int j = 0; j < TN; j++) T[(16 * i + e) * RS16 + 16 * j] = (int16_t)(acc[i][j][e] >> tsh);
    __syncthreads();
    // wave w copies tile row w: 16-byte chunk (pixel lane / 8 + 8 u, channels 8 (lane % 8) ..)
    if (oy < a.Ho) {
        const int16_t* T0 = (const int16_t*)smem + (wave * TW + (lane >> 3)) * RS16 + (lane & 7) * 8;
        int16_t* g = a.out16 + ((rowbase + ox0 + (lane >> 3)) * a.Nout + k0 + (lane & 7) * 8);
#pragma unroll
        for (int u = 0; u < TW / 8; u++)
            if ((lane >> 3) + 8 * u < vcols)
                *(int4*)(g + (int64_t)8 * u * a.Nout) = *(const int4*)&T0[8 * u * RS16];
    }
    if (tid == 0) {
        a.tshift[(int64_t)bx * gridDim.y + blockIdx.y] = (uint8_t)tsh;
        a.pmax[(int64_t)blockIdx.y * gridDim.x + blockIdx.x] = tmax;
    }
}

// ---------------------------------------------------------------------------
// 3x3 stride-1 convolution on v_mfma_i32_32x32x32_i8 (Ci % 64 == 0, Nout % 64
// == 0, dilation 1 or 2).  The 16x16x64 i8 MFMA issues at half the rate of the
// 32x32x32 form on gfx950, so this is the main path.
//
// A block owns a 16 x 32 output tile of one image and 64 output channels.  An
// A fragment is 32 pixels = 2 rows x 16 columns; wave w computes rows 4w..4w+3
// (four fragments) for all 64 channels (two B fragments): per tap and
// 32-channel half, 4 x 2 MFMAs from 6 LDS reads.  The halo (16 + 2 dh rows x
// 32 + 2 dw columns, one 64-channel chunk) and the 9 x 64 x 64 weight chunk
// are staged by direct-to-LDS loads.  Halo slots are swizzled by the column
// (slot = part ^ ((column >> 2) & 3)), which keeps any 16 consecutive pixels
// of a row conflict-free and leaves the swizzle unchanged by row offsets, so
// the nine taps need only three per-lane base addresses.
// ---------------------------------------------------------------------------
constexpr int kM32TH = 16, kM32TW = 32;
typedef int v16i_t __attribute__((ext_vector_type(16)));

// The 18 (tap, 32-channel half) steps of one 64-channel chunk.  Fragments of
// step k + 1 are read from LDS before the MFMAs of step k are issued (two
// register sets, scheduling barriers between the groups), so a single wave
// per SIMD keeps the matrix pipe fed instead of waiting on each LDS read.
template <int DH, int HC, int TM, int TN>
__device__ __forceinline__ void m32_taps(const int8_t* halo, const int8_t* w, const int (&abase)[3][2],
                                         const int (&bbase)[TN][2], v16i_t (&acc)[TM][TN], bool first)
{
    v4i fa[2][TM], fb[2][TN];
    auto load = [&](int k, int buf) {
        const int t = k >> 1, kh = k & 1, r = t / 3, s2 = t - (t / 3) * 3;
#pragma unroll
        for (int i = 0; i < TM; i++)          // fragment i: row pair 2 wave + i / 2, column group i % 2
            fa[buf][i] = *(const v4i*)&halo[abase[s2][kh] + (((i >> 1) * 2 + r * DH) * HC + 16 * (i & 1)) * 64];
#pragma unroll
        for (int j = 0; j < TN; j++) fb[buf][j] = *(const v4i*)&w[t * 4096 + bbase[j][kh]];
    };
    load(0, 0);
#pragma unroll
    for (int k = 0; k < 18; k++) {
        if (k + 1 < 18) load(k + 1, (k + 1) & 1);
        __builtin_amdgcn_sched_barrier(0);
        const int b = k & 1;
        if (k == 0 && first) {
#pragma unroll
            for (int i = 0; i < TM; i++)
#pragma unroll
                for (int j = 0; j < TN; j++)
                    acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fa[b][i], fb[b][j], (v16i_t){}, 0, 0, 0);
        } else {
#pragma unroll
            for (int i = 0; i < TM; i++)
#pragma unroll
                for (int j = 0; j < TN; j++)
                    acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fa[b][i], fb[b][j], acc[i][j], 0, 0, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
    }
}


template <int DH, int DW, int EPI>
__global__ __launch_bounds__(256, 2) void k_conv3x3_m32(HaloArgs a)
{
    constexpr int TH = kM32TH, TW = kM32TW, HR = TH + 2 * DH, HC = TW + 2 * DW;
    constexpr int TM = 4, TN = 2;
    constexpr int NHALO = HR * HC * 4;                      // 16-byte pieces
    constexpr int HBYTES = HR * HC * 64;
    extern __shared__ __attribute__((aligned(16))) int8_t smem[];
    int8_t* halo = smem;
    int8_t* wts = smem + HBYTES;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int nbx = gridDim.x;
    int bx = blockIdx.x;
    if ((nbx & 7) == 0) bx = (bx & 7) * (nbx >> 3) + (bx >> 3);
    const int tx = bx % a.tiles_x, t2 = bx / a.tiles_x;
    const int ty = t2 % a.tiles_y, n = t2 / a.tiles_y;
    const int oy0 = ty * TH, ox0 = tx * TW, k0 = blockIdx.y * 64;
    const int iy0 = oy0 - a.ph, ix0 = ox0 - a.pw;
    const int l32 = lane & 31, khalf = lane >> 5;          // fragment row, 16-byte half of a 32-byte k slice
    const int lr = l32 >> 4, lc = l32 & 15;                // row in the pair, column in the fragment

    // A base address of fragment (row pair 2 wave, column group 0) for column tap s and k half kh:
    // fragment (rp, cg), tap (r, s) adds ((2 rp + r DH) HC + 16 cg) * 64 (compile-time)
    int abase[3][2];
#pragma unroll
    for (int s2 = 0; s2 < 3; s2++)
#pragma unroll
        for (int kh = 0; kh < 2; kh++) {
            const int hc = lc + s2 * DW, part = 2 * kh + khalf;
            abase[s2][kh] = ((4 * wave + lr) * HC + hc) * 64 + ((part ^ ((hc >> 2) & 3)) << 4);
        }
    int bbase[TN][2];
#pragma unroll
    for (int j = 0; j < TN; j++)
#pragma unroll
        for (int kh = 0; kh < 2; kh++) {
            const int kk = 32 * j + l32, part = 2 * kh + khalf;
            bbase[j][kh] = kk * 64 + ((part ^ ((kk >> 2) & 3)) << 4);
        }
    // halo pieces: instruction k = wave + 4 u holds pixels 16 k .. 16 k + 15
    const int p0 = 16 * wave + (lane >> 2);
    const int hr0 = p0 / HC, hc0 = p0 - (p0 / HC) * HC;
    const int wkk = 16 * wave + (lane >> 2);
    const int wpart = (lane & 3) ^ ((wkk >> 2) & 3);
    const int8_t* wsrc = a.wmat + (int64_t)(k0 + wkk) * 9 * a.Ci + wpart * 16;

    v16i_t acc[TM][TN];
    const int nchunk = a.Ci / 64;
    uint64_t gmax = 0;
    for (int cc = 0; cc < nchunk; cc++) {
        if (cc) __syncthreads();                            // the previous chunk's reads are done
        {
            int hr = hr0, hc = hc0;
#pragma unroll
            for (int k = wave, u = 0; u < (NHALO / 64 + 4) / 4; u++, k += 4) {
                const int q = k * 64 + lane;
                if (q < NHALO) {
                    const int part = (q & 3) ^ ((hc >> 2) & 3);
                    const int iy = iy0 + hr, ix = ix0 + hc;
                    const bool v = (unsigned)iy < (unsigned)a.Hs && (unsigned)ix < (unsigned)a.Ws;
                    const void* g = v ? (const void*)(a.src + (((int64_t)n * a.Hs + iy) * a.Ws + ix) * a.Ci +
                                                      cc * 64 + part * 16)
                                      : (const void*)g_conv_zero;
                    dma16(g, halo + k * 1024);
                }
                hc += 64;
                while (hc >= HC) { hc -= HC; ++hr; }
            }
        }
#pragma unroll
        for (int j = 0; j < 9; j++)
            dma16(wsrc + (int64_t)j * a.Ci + cc * 64, wts + (wave + 4 * j) * 1024);
        if (EPI == EPI_Q8 && cc == 0) gmax = reduce_partials_u64(a.pmax, a.npmax);
        wait_vm<0>();
        __syncthreads();
        m32_taps<DH, HC, TM, TN>(halo, wts, abase, bbase, acc, cc == 0);
    }

    // acc[i][j][v]: fragment i (rows 4 wave + 2 (i / 2) + q / 16, columns 16 (i % 2) + q % 16 with
    // q = 8 (v / 4) + 4 khalf + v % 4), channel k0 + 32 j + l32
    auto px_row = [&](int i, int v) { return 4 * wave + 2 * (i >> 1) + ((8 * (v >> 2) + 4 * khalf + (v & 3)) >> 4); };
    auto px_col = [&](int i, int v) { return 16 * (i & 1) + ((8 * (v >> 2) + 4 * khalf + (v & 3)) & 15); };
    const int vrows = a.Ho - oy0 < TH ? a.Ho - oy0 : TH;
    const int vcols = a.Wo - ox0 < TW ? a.Wo - ox0 : TW;
    if (EPI == EPI_RAW) {
#pragma unroll
        for (int i = 0; i < TM; i++)
#pragma unroll
            for (int v = 0; v < 16; v++) {
                const int ry = px_row(i, v), rx = px_col(i, v);
                if (ry < vrows && rx < vcols) {
                    const int64_t pix = ((int64_t)n * a.Ho + oy0 + ry) * a.Wo + ox0 + rx;
#pragma unroll
                    for (int j = 0; j < TN; j++) a.out[pix * a.Nout + k0 + 32 * j + l32] = acc[i][j][v];
                }
            }
        return;
    }
    if (EPI == EPI_MAX) {
        int32_t vmax = 0, vmin = 0;
        const bool full = vrows == TH && vcols == TW;
#pragma unroll
        for (int i = 0; i < TM; i++)
#pragma unroll
            for (int v = 0; v < 16; v++)
                if (full || (px_row(i, v) < vrows && px_col(i, v) < vcols)) {
                    vmax = max(vmax, max(acc[i][0][v], acc[i][1][v]));
                    vmin = min(vmin, min(acc[i][0][v], acc[i][1][v]));
                }
        const uint64_t bm = block_max_u64((uint32_t)max(vmax, -vmin));
        if (tid == 0) a.pmax[(int64_t)blockIdx.y * gridDim.x + blockIdx.x] = bm;
        return;
    }
    // EPI_Q8: final SQ codes with r = bitlen(global max) - 7, staged per pixel row of 64 codes
    const int rq = gmax ? (64 - __builtin_clzll(gmax)) - 7 : 0;
    if (blockIdx.x == 0 && blockIdx.y == 0 && tid == 0) *a.out_exp = *a.exp_a + *a.exp_b + rq;
    const int rs = rq > 0 ? rq - 1 : 0, ls = rq > 0 ? 0 : -rq;
    constexpr int RB8 = 64 + 16;
    __syncthreads();                                        // every wave is done with the halo
#pragma unroll
    for (int i = 0; i < TM; i++)
#pragma unroll
        for (int v = 0; v < 16; v++) {
            const int px = px_row(i, v) * TW + px_col(i, v);
#pragma unroll
            for (int j = 0; j < TN; j++) {
                const int32_t x = acc[i][j][v];
                int32_t c = rq > 0 ? ((x >> rs) + 1) >> 1 : x << ls;
                c = c > 127 ? 127 : (c < -127 ? -127 : c);
                smem[px * RB8 + 32 * j + l32] = (int8_t)c;
            }
        }
    __syncthreads();
    // 512 pixels x 4 chunks of 16 codes: thread -> chunk (pixel c / 4, part c % 4)
#pragma unroll
    for (int u = 0; u < TH * TW * 4 / 256; u++) {
        const int c = tid + 256 * u;
        const int px = c >> 2, part = c & 3;
        const int ry = px / TW, rx = px % TW;
        if (ry < vrows && rx < vcols)
            *(int4*)(a.out8 + ((((int64_t)n * a.Ho + oy0 + ry) * a.Wo + ox0 + rx) * a.Nout + k0 + part * 16)) =
                *(const int4*)&smem[px * RB8 + part * 16];
    }
}

// Persistent form of the 32x32 kernel (Ci = 64 or 128): weights of all chunks
// stay in LDS, the next (tile, chunk) halo streams into the second buffer
// while the current one runs its taps, and a block walks a contiguous run of
// tiles (neighbours share halo rows and sit on one XCD).  One block per CU.
template <int DH, int DW, int EPI>
__global__ __launch_bounds__(256, 1) void k_conv3x3_m32p(HaloArgs a)
{
    constexpr int TH = kM32TH, TW = kM32TW, HR = TH + 2 * DH, HC = TW + 2 * DW;
    constexpr int TM = 4, TN = 2;
    constexpr int NHALO = HR * HC * 4;
    constexpr int RB8 = 64 + 16;
    constexpr int HBUF = (HR * HC * 64 > TH * TW * RB8 ? HR * HC * 64 : TH * TW * RB8);
    extern __shared__ __attribute__((aligned(16))) int8_t smem[];
    const int nchunk = a.Ci / 64;
    int8_t* wts = smem;                                     // [nchunk][9][64][64]
    int8_t* hb = smem + nchunk * 36864;                     // two halo / staging buffers of HBUF bytes

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int G = gridDim.x;
    int b = blockIdx.x;
    if ((G & 7) == 0) b = (b & 7) * (G >> 3) + (b >> 3);
    const int ntiles = a.N * a.tiles_y * a.tiles_x;
    const int t_begin = (int)((int64_t)b * ntiles / G), t_end = (int)((int64_t)(b + 1) * ntiles / G);
    const int nunits = (t_end - t_begin) * nchunk;
    const int k0 = blockIdx.y * 64;
    const int l32 = lane & 31, khalf = lane >> 5;
    const int lr = l32 >> 4, lc = l32 & 15;

    int abase[3][2];
#pragma unroll
    for (int s2 = 0; s2 < 3; s2++)
#pragma unroll
        for (int kh = 0; kh < 2; kh++) {
            const int hc = lc + s2 * DW, part = 2 * kh + khalf;
            abase[s2][kh] = ((4 * wave + lr) * HC + hc) * 64 + ((part ^ ((hc >> 2) & 3)) << 4);
        }
    int bbase[TN][2];
#pragma unroll
    for (int j = 0; j < TN; j++)
#pragma unroll
        for (int kh = 0; kh < 2; kh++) {
            const int kk = 32 * j + l32, part = 2 * kh + khalf;
            bbase[j][kh] = kk * 64 + ((part ^ ((kk >> 2) & 3)) << 4);
        }
    const int p0 = 16 * wave + (lane >> 2);
    const int hr0 = p0 / HC, hc0 = p0 - (p0 / HC) * HC;

    auto tile_origin = [&](int t, int& n, int& oy0, int& ox0) {
        const int tx = t % a.tiles_x, t2 = t / a.tiles_x;
        oy0 = (t2 % a.tiles_y) * TH;
        n = t2 / a.tiles_y;
        ox0 = tx * TW;
    };
    auto issue_halo = [&](int u) {
        const int t = t_begin + u / nchunk, cc = u - (u / nchunk) * nchunk;
        int n, oy0, ox0;
        tile_origin(t, n, oy0, ox0);
        const int iy0 = oy0 - a.ph, ix0 = ox0 - a.pw;
        int8_t* dst = hb + (u & 1) * HBUF;
        int hr = hr0, hc = hc0;
#pragma unroll
        for (int k = wave, v = 0; v < (NHALO / 64 + 4) / 4; v++, k += 4) {
            const int q = k * 64 + lane;
            if (q < NHALO) {
                const int part = (q & 3) ^ ((hc >> 2) & 3);
                const int iy = iy0 + hr, ix = ix0 + hc;
                const bool ok = (unsigned)iy < (unsigned)a.Hs && (unsigned)ix < (unsigned)a.Ws;
                const void* g = ok ? (const void*)(a.src + (((int64_t)n * a.Hs + iy) * a.Ws + ix) * a.Ci + cc * 64 +
                                                   part * 16)
                                   : (const void*)g_conv_zero;
                dma16(g, dst + k * 1024);
            }
            hc += 64;
            while (hc >= HC) { hc -= HC; ++hr; }
        }
    };

    {
        const int wkk = 16 * wave + (lane >> 2);
        const int wpart = (lane & 3) ^ ((wkk >> 2) & 3);
        const int8_t* wsrc = a.wmat + (int64_t)(k0 + wkk) * 9 * a.Ci + wpart * 16;
        for (int cc = 0; cc < nchunk; cc++)
#pragma unroll
            for (int j = 0; j < 9; j++)
                dma16(wsrc + (int64_t)j * a.Ci + cc * 64, wts + cc * 36864 + (wave + 4 * j) * 1024);
    }
    if (nunits > 0) issue_halo(0);
    uint64_t gmax = 0;
    if (EPI == EPI_Q8) gmax = reduce_partials_u64(a.pmax, a.npmax);
    const int rq = gmax ? (64 - __builtin_clzll(gmax)) - 7 : 0;
    wait_vm<0>();
    __syncthreads();

    v16i_t acc[TM][TN];
    int32_t vmax = 0, vmin = 0;
    for (int u = 0; u < nunits; u++) {
        if (u + 1 < nunits) issue_halo(u + 1);
        const int cc = u - (u / nchunk) * nchunk;
        const int8_t* halo = hb + (u & 1) * HBUF;
        const int8_t* w = wts + cc * 36864;
        m32_taps<DH, HC, TM, TN>(halo, w, abase, bbase, acc, cc == 0);
        if (cc == nchunk - 1) {
            int n, oy0, ox0;
            tile_origin(t_begin + u / nchunk, n, oy0, ox0);
            const int vrows = a.Ho - oy0 < TH ? a.Ho - oy0 : TH;
            const int vcols = a.Wo - ox0 < TW ? a.Wo - ox0 : TW;
            auto px_row = [&](int i, int v) {
                return 4 * wave + 2 * (i >> 1) + ((8 * (v >> 2) + 4 * khalf + (v & 3)) >> 4);
            };
            auto px_col = [&](int i, int v) { return 16 * (i & 1) + ((8 * (v >> 2) + 4 * khalf + (v & 3)) & 15); };
            if (EPI == EPI_RAW) {
#pragma unroll
                for (int i = 0; i < TM; i++)
#pragma unroll
                    for (int v = 0; v < 16; v++) {
                        const int ry = px_row(i, v), rx = px_col(i, v);
                        if (ry < vrows && rx < vcols) {
                            const int64_t pix = ((int64_t)n * a.Ho + oy0 + ry) * a.Wo + ox0 + rx;
#pragma unroll
                            for (int j = 0; j < TN; j++) a.out[pix * a.Nout + k0 + 32 * j + l32] = acc[i][j][v];
                        }
                    }
            } else if (EPI == EPI_MAX) {
                const bool full = vrows == TH && vcols == TW;
#pragma unroll
                for (int i = 0; i < TM; i++)
#pragma unroll
                    for (int v = 0; v < 16; v++)
                        if (full || (px_row(i, v) < vrows && px_col(i, v) < vcols)) {
                            vmax = max(vmax, max(acc[i][0][v], acc[i][1][v]));
                            vmin = min(vmin, min(acc[i][0][v], acc[i][1][v]));
                        }
            } else {
                const int rs = rq > 0 ? rq - 1 : 0, ls = rq > 0 ? 0 : -rq;
                int8_t* T = hb + (u & 1) * HBUF;            // this unit's halo buffer, now free
                __syncthreads();                            // every wave is done reading it
#pragma unroll
                for (int i = 0; i < TM; i++)
#pragma unroll
                    for (int v = 0; v < 16; v++) {
                        const int px = px_row(i, v) * TW + px_col(i, v);
#pragma unroll
                        for (int j = 0; j < TN; j++) {
                            const int32_t x = acc[i][j][v];
                            int32_t c = rq > 0 ? ((x >> rs) + 1) >> 1 : x << ls;
                            c = c > 127 ? 127 : (c < -127 ? -127 : c);
                            T[px * RB8 + 32 * j + l32] = (int8_t)c;
                        }
                    }
                __syncthreads();
#pragma unroll
                for (int v = 0; v < TH * TW * 4 / 256; v++) {
                    const int c = tid + 256 * v;
                    const int px = c >> 2, part = c & 3;
                    const int ry = px / TW, rx = px % TW;
                    if (ry < vrows && rx < vcols)
                        *(int4*)(a.out8 + ((((int64_t)n * a.Ho + oy0 + ry) * a.Wo + ox0 + rx) * a.Nout + k0 +
                                           part * 16)) = *(const int4*)&T[px * RB8 + part * 16];
                }
            }
        }
        wait_vm<0>();                                       // the next unit's halo has landed
        __syncthreads();
    }
    if (EPI == EPI_MAX) {
        const uint64_t bm = block_max_u64((uint32_t)max(vmax, -vmin));
        if (tid == 0) a.pmax[(int64_t)blockIdx.y * gridDim.x + blockIdx.x] = bm;
    }
    if (EPI == EPI_Q8 && blockIdx.x == 0 && blockIdx.y == 0 && tid == 0) *a.out_exp = *a.exp_a + *a.exp_b + rq;
}

// ---------------------------------------------------------------------------
// Stem convolution for few input channels (C = 3: 3x3 stride 1, 7x7 stride 2),
// Nout % 64 == 0.  The reduction (tap, channel) of R S C <= 160 entries is
// padded to k-steps of 32 and fed to v_mfma_i32_32x32x32_i8: a lane's A
// operand is 16 (tap, channel) bytes of one output pixel gathered from an LDS
// halo of the input tile, the B operand (the weights, KRSC order = the same
// reduction order) stays in registers for the whole block.  A block owns 16 x
// 32 output pixels (wave w: rows 4w..4w+3, one 32-pixel fragment per row) and
// 64 output channels.  Epilogues as for the 3x3 kernels (raw sums, max pass,
// final codes).
// ---------------------------------------------------------------------------
template <int C, int R, int S, int ST, int EPI>
__global__ __launch_bounds__(256) void k_conv_stem(HaloArgs a)
{
    constexpr int TH = 16, TW = 32, KRED = R * S * C, NKS = (KRED + 31) / 32;
    constexpr int HROWS = (TH - 1) * ST + R, HCOLS = (TW - 1) * ST + S;
    constexpr int HBYTES = (HROWS * HCOLS * C + 15) & ~15;
    constexpr int RB8 = 64 + 16;
    __shared__ __attribute__((aligned(16))) int8_t smem[HBYTES > TH * TW * RB8 ? HBYTES : TH * TW * RB8];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int l32 = lane & 31, h = lane >> 5;
    const int tx = blockIdx.x % a.tiles_x, t2 = blockIdx.x / a.tiles_x;
    const int ty = t2 % a.tiles_y, n = t2 / a.tiles_y;
    const int oy0 = ty * TH, ox0 = tx * TW, k0 = blockIdx.y * 64;
    const int iy0 = oy0 * ST - a.ph, ix0 = ox0 * ST - a.pw;

    // halo: rows iy0 .. iy0 + HROWS - 1, columns ix0 .., all C channels (zero outside the
    // image); every load of a thread is issued before its first LDS store
    {
        constexpr int NH = HROWS * HCOLS * C, PER = (NH + 255) / 256;
        int8_t hv[PER];
#pragma unroll
        for (int u = 0; u < PER; u++) {
            const int i = tid + 256 * u;
            const int hr = i / (HCOLS * C), rem = i - hr * (HCOLS * C);
            const int hc = rem / C, c = rem - hc * C;
            const int iy = iy0 + hr, ix = ix0 + hc;
            const bool v = i < NH && (unsigned)iy < (unsigned)a.Hs && (unsigned)ix < (unsigned)a.Ws;
            hv[u] = v ? a.src[(((int64_t)n * a.Hs + iy) * a.Ws + ix) * C + c] : (int8_t)0;
        }
#pragma unroll
        for (int u = 0; u < PER; u++)
            if (tid + 256 * u < NH) smem[tid + 256 * u] = hv[u];
    }
    uint64_t gmax = 0;
    if (EPI == EPI_Q8) gmax = reduce_partials_u64(a.pmax, a.npmax);
    // B: weights of channels k0 + 32 j + l32, reduction bytes 32 ks + 16 h + b (zero past KRED)
    v4i fb[NKS][2];
#pragma unroll
    for (int ks = 0; ks < NKS; ks++)
#pragma unroll
        for (int j = 0; j < 2; j++) {
            uint32_t wv[4] = {0, 0, 0, 0};
            const int8_t* wr = a.wmat + (int64_t)(k0 + 32 * j + l32) * KRED;
#pragma unroll
            for (int b = 0; b < 16; b++) {
                const int k = 32 * ks + 16 * h + b;
                if (k < KRED) wv[b >> 2] |= (uint32_t)(uint8_t)wr[k] << (8 * (b & 3));
            }
            fb[ks][j] = (v4i){(int)wv[0], (int)wv[1], (int)wv[2], (int)wv[3]};
        }
    // A gather offsets (relative to the pixel's halo origin) of this lane's 16 reduction bytes
    int aoff[NKS][16];
#pragma unroll
    for (int ks = 0; ks < NKS; ks++)
#pragma unroll
        for (int b = 0; b < 16; b++) {
            const int k = 32 * ks + 16 * h + b;
            const int tap = k / C, c = k - (k / C) * C, r = tap / S, s2 = tap - (tap / S) * S;
            aoff[ks][b] = k < KRED ? (r * HCOLS + s2) * C + c : -1;
        }
    __syncthreads();

    typedef int v16i __attribute__((ext_vector_type(16)));
    v16i acc[4][2];
#pragma unroll
    for (int f = 0; f < 4; f++) {
        const int pbase = ((4 * wave + f) * ST * HCOLS + l32 * ST) * C;
#pragma unroll
        for (int ks = 0; ks < NKS; ks++) {
            uint32_t av[4] = {0, 0, 0, 0};
#pragma unroll
            for (int b = 0; b < 16; b++)
                if (aoff[ks][b] >= 0) av[b >> 2] |= (uint32_t)(uint8_t)smem[pbase + aoff[ks][b]] << (8 * (b & 3));
            const v4i fa = (v4i){(int)av[0], (int)av[1], (int)av[2], (int)av[3]};
#pragma unroll
            for (int j = 0; j < 2; j++)
                acc[f][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fa, fb[ks][j], ks ? acc[f][j] : (v16i){}, 0, 0, 0);
        }
    }

    // acc[f][j][v]: output row 4 wave + f, column 8 (v / 4) + 4 h + v % 4, channel k0 + 32 j + l32
    const int vrows = a.Ho - oy0 < TH ? a.Ho - oy0 : TH;
    const int vcols = a.Wo - ox0 < TW ? a.Wo - ox0 : TW;
    auto colof = [&](int v) { return 8 * (v >> 2) + 4 * h + (v & 3); };
    if (EPI == EPI_RAW) {
#pragma unroll
        for (int f = 0; f < 4; f++)
#pragma unroll
            for (int v = 0; v < 16; v++)
                if (4 * wave + f < vrows && colof(v) < vcols) {
                    const int64_t pix = ((int64_t)n * a.Ho + oy0 + 4 * wave + f) * a.Wo + ox0 + colof(v);
#pragma unroll
                    for (int j = 0; j < 2; j++) a.out[pix * a.Nout + k0 + 32 * j + l32] = acc[f][j][v];
                }
        return;
    }
    if (EPI == EPI_MAX) {
        int32_t vmax = 0, vmin = 0;
#pragma unroll
        for (int f = 0; f < 4; f++)
#pragma unroll
            for (int v = 0; v < 16; v++)
                if (4 * wave + f < vrows && colof(v) < vcols) {
                    vmax = max(vmax, max(acc[f][0][v], acc[f][1][v]));
                    vmin = min(vmin, min(acc[f][0][v], acc[f][1][v]));
                }
        const uint64_t bm = block_max_u64((uint32_t)max(vmax, -vmin));
        if (tid == 0) a.pmax[(int64_t)blockIdx.y * gridDim.x + blockIdx.x] = bm;
        return;
    }
    const int rq = gmax ? (64 - __builtin_clzll(gmax)) - 7 : 0;
    if (blockIdx.x == 0 && blockIdx.y == 0 && tid == 0) *a.out_exp = *a.exp_a + *a.exp_b + rq;
    const int rs = rq > 0 ? rq - 1 : 0, ls = rq > 0 ? 0 : -rq;
    __syncthreads();                                         // the halo is no longer read
#pragma unroll
    for (int f = 0; f < 4; f++)
#pragma unroll
        for (int v = 0; v < 16; v++) {
            const int px = (4 * wave + f) * TW + colof(v);
#pragma unroll
            for (int j = 0; j < 2; j++) {
                const int32_t x = acc[f][j][v];
                int32_t c = rq > 0 ? ((x >> rs) + 1) >> 1 : x << ls;
                c = c > 127 ? 127 : (c < -127 ? -127 : c);
                smem[px * RB8 + 32 * j + l32] = (int8_t)c;
            }
        }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < TH * TW * 4 / 256; u++) {
        const int c = tid + 256 * u;
        const int px = c >> 2, part = c & 3;
        const int ry = px / TW, rx = px % TW;
        if (ry < vrows && rx < vcols)
            *(int4*)(a.out8 + ((((int64_t)n * a.Ho + oy0 + ry) * a.Wo + ox0 + rx) * a.Nout + k0 + part * 16)) =
                *(const int4*)&smem[px * RB8 + part * 16];
    }
}

// shapes of the stem kernel: C = 3 with 3x3 / stride 1 or 7x7 / stride 2, no dilation
int stem_kind(int64_t C, int R, int S, int sh, int sw, int dh, int dw, int64_t Nout)
{
    if (C != 3 || dh != 1 || dw != 1 || Nout % 64 != 0) return 0;
    if (R == 3 && S == 3 && sh == 1 && sw == 1) return 1;
    if (R == 7 && S == 7 && sh == 2 && sw == 2) return 2;
    return 0;
}

template <int R, int ST, int EPI>
int launch_stem_t(const HaloArgs& a, int kid, hipStream_t s)
{
    dim3 grid((unsigned)(a.N * a.tiles_y * a.tiles_x), (unsigned)(a.Nout / 64));
    ISEG_TIMED_LAUNCH(kid, s, (k_conv_stem<3, R, R, ST, EPI>), grid, dim3(256), 0, s, a);
    return launch_ok();
}

int launch_stem(int kind, HaloArgs a, int epi, int kid, hipStream_t s)
{
    a.tiles_y = (int)ceil_div64(a.Ho, 16);
    a.tiles_x = (int)ceil_div64(a.Wo, 32);
    if (kind == 1) {
        if (epi == EPI_RAW) return launch_stem_t<3, 1, EPI_RAW>(a, kid, s);
        if (epi == EPI_MAX) return launch_stem_t<3, 1, EPI_MAX>(a, kid, s);
        return launch_stem_t<3, 1, EPI_Q8>(a, kid, s);
    }
    if (epi == EPI_RAW) return launch_stem_t<7, 2, EPI_RAW>(a, kid, s);
    if (epi == EPI_MAX) return launch_stem_t<7, 2, EPI_MAX>(a, kid, s);
    return launch_stem_t<7, 2, EPI_Q8>(a, kid, s);
}

struct M32Plan {
    bool ok;
    int tiles_y, tiles_x;
    size_t lds;
    bool persist;                 // weights resident, double-buffered halos
    int G;                        // persistent blocks per 64-channel group
    size_t plds;
};

M32Plan m32_plan(int64_t N, int64_t Ho, int64_t Wo, int64_t Ci, int64_t Nout, int R, int S, int sh, int sw, int dh,
                 int dw)
{
    M32Plan p{};
    p.ok = N > 0 && R == 3 && S == 3 && sh == 1 && sw == 1 && dh >= 1 && dh <= 2 && dw >= 1 && dw <= 2 &&
           Ci % 64 == 0 && Ci <= 128 && Nout % 64 == 0 && N * Ho * Wo < ((int64_t)1 << 31);
    if (!p.ok) return p;
    p.tiles_y = (int)ceil_div64(Ho, kM32TH);
    p.tiles_x = (int)ceil_div64(Wo, kM32TW);
    const size_t halo = (size_t)(kM32TH + 2 * dh) * (kM32TW + 2 * dw) * 64;
    p.lds = halo + 9 * 64 * 64;
    const size_t stage = (size_t)kM32TH * kM32TW * 80;
    if (p.lds < stage) p.lds = stage;
    p.ok = N * p.tiles_y * p.tiles_x < ((int64_t)1 << 31);
    const int64_t ntiles = N * p.tiles_y * p.tiles_x, groups = Nout / 64;
    const size_t hbuf = halo > stage ? halo : stage;
    p.plds = (size_t)(Ci / 64) * 36864 + 2 * hbuf;
    int64_t G = 256 / groups;
    if (G < 8) G = 8;
    if (G > ntiles) G = ntiles;
    p.G = (int)G;
    p.persist = false;   // measured slower than two resident blocks per CU at these sizes
    (void)ntiles;
    return p;
}

template <int DH, int DW, int EPI>
int launch_m32_t(const M32Plan& p, const HaloArgs& a, int kid, hipStream_t s)
{
    if (p.persist) {
        dim3 grid((unsigned)p.G, (unsigned)(a.Nout / 64));
        if (!lds_limit((const void*)k_conv3x3_m32p<DH, DW, EPI>, (size_t)p.plds))
            return ISEG_ERR_DEVICE;
        ISEG_TIMED_LAUNCH(kid, s, (k_conv3x3_m32p<DH, DW, EPI>), grid, dim3(256), p.plds, s, a);
        return launch_ok();
    }
    dim3 grid((unsigned)(a.N * p.tiles_y * p.tiles_x), (unsigned)(a.Nout / 64));
    if (!lds_limit((const void*)k_conv3x3_m32<DH, DW, EPI>, (size_t)p.lds))
        return ISEG_ERR_DEVICE;
    ISEG_TIMED_LAUNCH(kid, s, (k_conv3x3_m32<DH, DW, EPI>), grid, dim3(256), p.lds, s, a);
    return launch_ok();
}

template <int EPI>
int launch_m32_e(const M32Plan& p, const HaloArgs& a, int kid, hipStream_t s)
{
    if (a.dh == 1 && a.dw == 1) return launch_m32_t<1, 1, EPI>(p, a, kid, s);
    if (a.dh == 2 && a.dw == 2) return launch_m32_t<2, 2, EPI>(p, a, kid, s);
    if (a.dh == 1) return launch_m32_t<1, 2, EPI>(p, a, kid, s);
    return launch_m32_t<2, 1, EPI>(p, a, kid, s);
}

int launch_m32(const M32Plan& p, HaloArgs a, int epi, int kid, hipStream_t s)
{
    a.tiles_y = p.tiles_y;
    a.tiles_x = p.tiles_x;
    if (epi == EPI_RAW) return launch_m32_e<EPI_RAW>(p, a, kid, s);
    if (epi == EPI_MAX) return launch_m32_e<EPI_MAX>(p, a, kid, s);
    return launch_m32_e<EPI_Q8>(p, a, kid, s);
}

// Q8 through the 32x32 kernel: max pass, then the final-code pass
int m32_q8(const M32Plan& p, HaloArgs h, int kid, const int32_t* exp_a, const int32_t* exp_b, int8_t* out,
           int32_t* out_exp, uint64_t* pmax, hipStream_t s)
{
    int rc;
    h.pmax = pmax;
    h.npmax = p.persist ? (int64_t)p.G * (h.Nout / 64) : (int64_t)h.N * p.tiles_y * p.tiles_x * (h.Nout / 64);
    if ((rc = launch_m32(p, h, EPI_MAX, kid, s))) return rc;
    h.out8 = out; h.exp_a = exp_a; h.exp_b = exp_b; h.out_exp = out_exp;
    return launch_m32(p, h, EPI_Q8, kid, s);
}

// ---------------------------------------------------------------------------
// Persistent variant (Ci = 64 or 128): a block keeps its 64 output channels'
// weights for all chunks resident in LDS and walks a contiguous run of tiles;
// the input halo of the next (tile, chunk) streams into the second of two
// buffers while the current one runs its nine taps, so the loads hide behind
// the MFMAs.  The final-code epilogue stages a tile's codes in the halo buffer
// it has just finished with.  Blocks are numbered so that neighbouring tiles
// (which share halo rows) run on one XCD.
// ---------------------------------------------------------------------------
template <int TW, int EPI>
__global__ __launch_bounds__(256) void k_conv3x3_persist(HaloArgs a)
{
    constexpr int TH = kHaloTH, TM = TW / 16, TN = 4;
    extern __shared__ __attribute__((aligned(16))) int8_t smem[];
    const int HR = TH + 2 * a.dh, HC = TW + 2 * a.dw;
    const int nhalo = HR * HC * 4;                        // 16-byte pieces per halo
    const int nchunk = a.Ci / 64;
    int8_t* wts = smem;                                   // [nchunk][9][64][64]
    int8_t* hbuf0 = smem + nchunk * 36864;
    const int hbytes = HR * HC * 64;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int G = gridDim.x;
    int b = blockIdx.x;
    if ((G & 7) == 0) b = (b & 7) * (G >> 3) + (b >> 3);
    const int ntiles = a.N * a.tiles_y * a.tiles_x;
    const int t_begin = (int)((int64_t)b * ntiles / G), t_end = (int)((int64_t)(b + 1) * ntiles / G);
    const int nunits = (t_end - t_begin) * nchunk;
    const int k0 = blockIdx.y * 64;
    const int lrow = lane & 15, lpart = lane >> 4;

    int aaddr[9];
#pragma unroll
    for (int r = 0; r < 3; r++)
#pragma unroll
        for (int s2 = 0; s2 < 3; s2++) {
            const int p = (wave + r * a.dh) * HC + lrow + s2 * a.dw;
            aaddr[r * 3 + s2] = p * 64 + ((lpart ^ ((p >> 2) & 3)) << 4);
        }
    int baddr[TN];
#pragma unroll
    for (int j = 0; j < TN; j++) {
        const int kk = 16 * j + lrow;
        baddr[j] = kk * 64 + ((lpart ^ ((kk >> 2) & 3)) << 4);
    }
    const int p0 = 16 * wave + (lane >> 2);
    const int hr0 = p0 / HC, hc0 = p0 - (p0 / HC) * HC;

    // tile t -> (image, tile row, tile column)
    auto tile_origin = [&](int t, int& n, int& oy0, int& ox0) {
        const int tx = t % a.tiles_x, t2 = t / a.tiles_x;
        oy0 = (t2 % a.tiles_y) * TH;
        n = t2 / a.tiles_y;
        ox0 = tx * TW;
    };
    auto issue_halo = [&](int u) {
        const int t = t_begin + u / nchunk, cc = u - (u / nchunk) * nchunk;
        int n, oy0, ox0;
        tile_origin(t, n, oy0, ox0);
        const int iy0 = oy0 - a.ph, ix0 = ox0 - a.pw;
        int8_t* dst = hbuf0 + (u & 1) * hbytes;
        int hr = hr0, hc = hc0;
        for (int k = wave; k * 64 < nhalo; k += 4) {
            const int q = k * 64 + lane;
            if (q < nhalo) {
                const int p = q >> 2;
                const int part = (q & 3) ^ ((p >> 2) & 3);
                const int iy = iy0 + hr, ix = ix0 + hc;
                const bool v = (unsigned)iy < (unsigned)a.Hs && (unsigned)ix < (unsigned)a.Ws;
                const void* g = v ? (const void*)(a.src + (((int64_t)n * a.Hs + iy) * a.Ws + ix) * a.Ci + cc * 64 +
                                                  part * 16)
                                  : (const void*)g_conv_zero;
                dma16(g, dst + k * 1024);
            }
            hc += 64;
            while (hc >= HC) { hc -= HC; ++hr; }
        }
    };

    // prologue: every chunk's weights, the first halo, the global max (second pass)
    {
        const int wkk = 16 * wave + (lane >> 2);
        const int wpart = (lane & 3) ^ ((wkk >> 2) & 3);
        const int8_t* wsrc = a.wmat + (int64_t)(k0 + wkk) * 9 * a.Ci + wpart * 16;
        for (int cc = 0; cc < nchunk; cc++)
#pragma unroll
            for (int j = 0; j < 9; j++)
                dma16(wsrc + (int64_t)j * a.Ci + cc * 64, wts + cc * 36864 + (wave + 4 * j) * 1024);
    }
    if (nunits > 0) issue_halo(0);
    uint64_t gmax = 0;
    if (EPI == EPI_Q8) gmax = reduce_partials_u64(a.pmax, a.npmax);
    wait_vm<0>();
    __syncthreads();

    int32_t vmax = 0, vmin = 0;                           // max pass: running extremes
    v4i acc[TM][TN];
    for (int u = 0; u < nunits; u++) {
        if (u + 1 < nunits) issue_halo(u + 1);
        const int cc = u - (u / nchunk) * nchunk;
        const int8_t* halo = hbuf0 + (u & 1) * hbytes;
        const int8_t* w = wts + cc * 36864;
#pragma unroll
        for (int t = 0; t < 9; t++) {
            v4i fa[TM], fb[TN];
#pragma unroll
            for (int i = 0; i < TM; i++) fa[i] = *(const v4i*)&halo[aaddr[t] + 1024 * i];
#pragma unroll
            for (int j = 0; j < TN; j++) fb[j] = *(const v4i*)&w[t * 4096 + baddr[j]];
            if (t == 0 && cc == 0) {
#pragma unroll
                for (int i = 0; i < TM; i++)
#pragma unroll
                    for (int j = 0; j < TN; j++)
                        acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[i], fb[j], (v4i){0, 0, 0, 0}, 0, 0, 0);
            } else {
#pragma unroll
                for (int i = 0; i < TM; i++)
#pragma unroll
                    for (int j = 0; j < TN; j++)
                        acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[i], fb[j], acc[i][j], 0, 0, 0);
            }
        }
        if (cc == nchunk - 1) {
            int n, oy0, ox0;
            tile_origin(t_begin + u / nchunk, n, oy0, ox0);
            const int oy = oy0 + wave;
            const int vcols = a.Wo - ox0 < TW ? a.Wo - ox0 : TW;
            const int64_t rowbase = ((int64_t)n * a.Ho + oy) * a.Wo;
            if (EPI == EPI_RAW) {
                if (oy < a.Ho) {
#pragma unroll
                    for (int i = 0; i < TM; i++)
#pragma unroll
                        for (int e = 0; e < 4; e++)
                            if (16 * i + 4 * lpart + e < vcols) {
#pragma unroll
                                for (int j = 0; j < TN; j++)
                                    a.out[(rowbase + ox0 + 16 * i + 4 * lpart + e) * a.Nout + k0 + 16 * j + lrow] =
                                        acc[i][j][e];
                            }
                }
            } else if (EPI == EPI_MAX) {
                if (oy < a.Ho) {
#pragma unroll
                    for (int i = 0; i < TM; i++)
#pragma unroll
                        for (int e = 0; e < 4; e++)
                            if (16 * i + 4 * lpart + e < vcols) {
#pragma unroll
                                for (int j = 0; j < TN; j += 2) {
                                    vmax = max(vmax, max(acc[i][j][e], acc[i][j + 1][e]));
                                    vmin = min(vmin, min(acc[i][j][e], acc[i][j + 1][e]));
                                }
                            }
                }
            } else {                                      // EPI_Q8
                const int r = gmax ? (64 - __builtin_clzll(gmax)) - 7 : 0;
                const int rs = r > 0 ? r - 1 : 0, ls = r > 0 ? 0 : -r;
                constexpr int RB8 = 64 + 16;
                int8_t* T = (int8_t*)halo + (wave * TW + 4 * lpart) * RB8 + lrow;
                __syncthreads();                          // every wave is done reading this halo
#pragma unroll
                for (int i = 0; i < TM; i++)
#pragma unroll
                    for (int e = 0; e < 4; e++)
#pragma unroll
                        for (int j = 0; j < TN; j++) {
                            const int32_t v = acc[i][j][e];
                            int32_t c = r > 0 ? ((v >> rs) + 1) >> 1 : v << ls;
                            c = c > 127 ? 127 : (c < -127 ? -127 : c);
                            T[(16 * i + e) * RB8 + 16 * j] = (int8_t)c;
                        }
                __syncthreads();
                if (oy < a.Ho) {
                    const int8_t* T0 = halo + (wave * TW + (lane >> 2)) * RB8 + (lane & 3) * 16;
                    int8_t* g = a.out8 + ((rowbase + ox0 + (lane >> 2)) * a.Nout + k0 + (lane & 3) * 16);
#pragma unroll
                    for (int u2 = 0; u2 < TW / 16; u2++)
                        if ((lane >> 2) + 16 * u2 < vcols)
                            *(int4*)(g + (int64_t)16 * u2 * a.Nout) = *(const int4*)&T0[16 * u2 * RB8];
                }
            }
        }
        wait_vm<0>();                                     // the next unit's halo has landed
        __syncthreads();
    }
    if (EPI == EPI_MAX) {
        const uint64_t bm = block_max_u64((uint32_t)max(vmax, -vmin));
        if (tid == 0) a.pmax[(int64_t)blockIdx.y * gridDim.x + blockIdx.x] = bm;
    }
    if (EPI == EPI_Q8 && blockIdx.x == 0 && blockIdx.y == 0 && tid == 0) {
        const int r = gmax ? (64 - __builtin_clzll(gmax)) - 7 : 0;
        *a.out_exp = *a.exp_a + *a.exp_b + r;
    }
}

struct PersistPlan {
    bool ok;
    int TW, tiles_y, tiles_x, G;
    size_t lds;
};

PersistPlan persist_plan(int64_t N, int64_t Ho, int64_t Wo, int64_t Ci, int64_t Nout, int R, int S, int sh, int sw,
                         int dh, int dw)
{
    PersistPlan p{};
    p.ok = N > 0 && R == 3 && S == 3 && sh == 1 && sw == 1 && dh <= 2 && dw <= 2 && (Ci == 64 || Ci == 128) &&
           Nout % 64 == 0 && N * Ho * Wo < ((int64_t)1 << 31);
    if (!p.ok) return p;
    p.TW = (Ci == 64 && Wo % 112 == 0) ? 112 : 64;
    p.tiles_y = (int)ceil_div64(Ho, kHaloTH);
    p.tiles_x = (int)ceil_div64(Wo, p.TW);
    const int64_t ntiles = N * p.tiles_y * p.tiles_x;
    const int64_t halo = (int64_t)(kHaloTH + 2 * dh) * (p.TW + 2 * dw) * 64;
    p.lds = (size_t)((Ci / 64) * 36864 + 2 * halo);
    const int64_t groups = Nout / 64;
    int64_t G = 256 / groups;
    if (G < 8) G = 8;
    if (G > ntiles) G = ntiles;
    p.G = (int)G;
    p.ok = ntiles < ((int64_t)1 << 31) && p.lds <= 160 * 1024 &&
           (int64_t)kHaloTH * p.TW * 80 <= halo;        // code staging fits in a halo buffer
    return p;
}

template <int TW, int EPI>
int launch_persist_t(const PersistPlan& p, const HaloArgs& a, int kid, hipStream_t s)
{
    dim3 grid((unsigned)p.G, (unsigned)(a.Nout / 64));
    if (!lds_limit((const void*)k_conv3x3_persist<TW, EPI>, (size_t)p.lds))
        return ISEG_ERR_DEVICE;
    ISEG_TIMED_LAUNCH(kid, s, (k_conv3x3_persist<TW, EPI>), grid, dim3(256), p.lds, s, a);
    return launch_ok();
}

int launch_persist(const PersistPlan& p, HaloArgs a, int epi, int kid, hipStream_t s)
{
    a.tiles_y = p.tiles_y;
    a.tiles_x = p.tiles_x;
    if (p.TW == 112) {
        if (epi == EPI_RAW) return launch_persist_t<112, EPI_RAW>(p, a, kid, s);
        if (epi == EPI_MAX) return launch_persist_t<112, EPI_MAX>(p, a, kid, s);
        return launch_persist_t<112, EPI_Q8>(p, a, kid, s);
    }
    if (epi == EPI_RAW) return launch_persist_t<64, EPI_RAW>(p, a, kid, s);
    if (epi == EPI_MAX) return launch_persist_t<64, EPI_MAX>(p, a, kid, s);
    return launch_persist_t<64, EPI_Q8>(p, a, kid, s);
}

// Q8 through the persistent kernel: max pass, then the final-code pass
int persist_q8(const PersistPlan& p, HaloArgs h, int kid, const int32_t* exp_a, const int32_t* exp_b, int8_t* out,
               int32_t* out_exp, uint64_t* pmax, hipStream_t s)
{
    int rc;
    h.pmax = pmax;
    h.npmax = (int64_t)p.G * (h.Nout / 64);
    if ((rc = launch_persist(p, h, EPI_MAX, kid, s))) return rc;
    h.out8 = out; h.exp_a = exp_a; h.exp_b = exp_b; h.out_exp = out_exp;
    return launch_persist(p, h, EPI_Q8, kid, s);
}


// the halo kernel covers 3x3 filters at stride 1, dilation <= 2, Ci and Nout
// multiples of 64, 16-byte aligned operands
struct HaloPlan {
    bool ok;
    int TW;
    int tiles_y, tiles_x;
    size_t lds;
};

HaloPlan halo_plan(int64_t N, int64_t Ho, int64_t Wo, int64_t Ci, int64_t Nout, int R, int S, int sh, int sw,
                   int dh, int dw)
{
    HaloPlan p{};
    p.ok = N > 0 && R == 3 && S == 3 && sh == 1 && sw == 1 && dh <= 2 && dw <= 2 && Ci % 64 == 0 &&
           Nout % 64 == 0 && N * Ho * Wo < ((int64_t)1 << 31);
    if (!p.ok) return p;
    // widest tile without a ragged column tile when the width allows it
    p.TW = (Wo % 112 == 0) ? 112 : 64;
    p.tiles_y = (int)ceil_div64(Ho, kHaloTH);
    p.tiles_x = (int)ceil_div64(Wo, p.TW);
    p.lds = halo_lds_bytes(p.TW, dh, dw);
    p.ok = N * p.tiles_y * p.tiles_x < ((int64_t)1 << 31);
    return p;
}

size_t halo_staged_ws_bytes(const HaloPlan& p, int64_t N, int64_t Ho, int64_t Wo, int64_t Nout)
{
    return align256((size_t)(N * Ho * Wo * Nout) * 2) +
           align256((size_t)(N * p.tiles_y * p.tiles_x * (Nout / 64)));
}

template <int TW, int EPI>
int launch_halo_t(const HaloPlan& p, const HaloArgs& a, int kid, hipStream_t s)
{
    dim3 grid((unsigned)(a.N * p.tiles_y * p.tiles_x), (unsigned)(a.Nout / 64));
    if (!lds_limit((const void*)k_conv3x3_halo<TW, EPI>, (size_t)p.lds))
        return ISEG_ERR_DEVICE;
    ISEG_TIMED_LAUNCH(kid, s, (k_conv3x3_halo<TW, EPI>), grid, dim3(256), p.lds, s, a);
    return launch_ok();
}

int launch_halo(const HaloPlan& p, HaloArgs a, int epi, int kid, hipStream_t s)
{
    a.tiles_y = p.tiles_y;
    a.tiles_x = p.tiles_x;
    if (p.TW == 112) {
        switch (epi) {
        case EPI_RAW: return launch_halo_t<112, EPI_RAW>(p, a, kid, s);
        case EPI_STAGE16: return launch_halo_t<112, EPI_STAGE16>(p, a, kid, s);
        case EPI_MAX: return launch_halo_t<112, EPI_MAX>(p, a, kid, s);
        default: return launch_halo_t<112, EPI_Q8>(p, a, kid, s);
        }
    }
    switch (epi) {
    case EPI_RAW: return launch_halo_t<64, EPI_RAW>(p, a, kid, s);
    case EPI_STAGE16: return launch_halo_t<64, EPI_STAGE16>(p, a, kid, s);
    case EPI_MAX: return launch_halo_t<64, EPI_MAX>(p, a, kid, s);
    default: return launch_halo_t<64, EPI_Q8>(p, a, kid, s);
    }
}

// Q8 output through the halo kernel: for short reductions (Ci <= kTwoPassMaxCi)
// a max-only pass and a recomputing pass that writes final codes, else int16
// staging plus a requant pass.  The recompute costs 9 Ci MACs per output while
// staging moves 4 more bytes per output through HBM.
constexpr int kTwoPassMaxCi = 128;

int halo_q8(const HaloPlan& p, HaloArgs h, int kid, const int32_t* exp_a, const int32_t* exp_b, int8_t* out,
            int32_t* out_exp, unsigned long long* maxp, uint64_t* pmax, int64_t rows, hipStream_t s)
{
    int rc;
    h.pmax = pmax;
    h.npmax = (int64_t)h.N * p.tiles_y * p.tiles_x * (h.Nout / 64);
    if (h.Ci <= kTwoPassMaxCi) {
        if ((rc = launch_halo(p, h, EPI_MAX, kid, s))) return rc;
        h.out8 = out; h.exp_a = exp_a; h.exp_b = exp_b; h.out_exp = out_exp;
        return launch_halo(p, h, EPI_Q8, kid, s);
    }
    if ((rc = launch_halo(p, h, EPI_STAGE16, kid, s))) return rc;
    (void)maxp;
    StageMap sm{0, 64, h.Ho, h.Wo, kHaloTH, p.TW, p.tiles_y, p.tiles_x};
    return launch_requant_staged16(h.out16, h.tshift, rows, h.Nout, sm, exp_a, exp_b, 8, out, out_exp, nullptr, s,
                                   pmax, h.npmax);
}

// the direct-to-LDS kernel covers Ci % 64 == 0, Nout % 64 == 0, 16-byte
// aligned operands and fewer than 2^31 rows; its int16-staged output is used
// whenever the result is requantized
bool igemm_dma_ok(const IgemmArgs& a)
{
    return a.Mrows > 0 && a.Mrows < ((int64_t)1 << 31) && a.Ci % 64 == 0 && a.Nout % 64 == 0 && a.R * a.S <= 64 &&
           (((uintptr_t)a.src | (uintptr_t)a.wmat) & 15) == 0;
}
size_t staged_ws_bytes(int64_t rows, int64_t cols)
{
    return align256((size_t)(rows * cols) * 2) + align256((size_t)(ceil_div64(rows, 128) * ceil_div64(cols, 64)));
}

// Direct-to-LDS GEMM plan.  Short reductions (Kred <= 256) with final codes
// take two passes over 128-row tiles (max partials, then recomputed codes):
// cheaper than staging when each output costs few MACs.  Otherwise ISEG_IGEMM_BM-row
// tiles, with the reduction split over gridDim.z when the output tiles alone
// would leave CUs idle and the reduction is long (at least 32 steps of 64 per
// split: a split costs a reduce and an int32 requant pass).  256-row tiles
// (ISEG_IGEMM_BM) cut LDS and L2 traffic per MAC by a quarter but need more
// registers than two waves per SIMD allow; 128-row tiles measure faster.
#ifndef ISEG_IGEMM_BM
#define ISEG_IGEMM_BM 128
#endif
#ifndef ISEG_IGEMM_PIPE
#define ISEG_IGEMM_PIPE 1
#endif
#ifndef ISEG_IGEMM_SPLIT_BLOCKS
#define ISEG_IGEMM_SPLIT_BLOCKS 512       // split until this many blocks (0: never split)
#endif
constexpr int kTwoPassMaxKred = 256;
constexpr int kMaxSplits = 8;
struct DmaPlan {
    bool two_pass;
    int bm, bn, splits;
};
DmaPlan dma_plan(int64_t Mrows, int32_t Nout, int32_t Kred, bool q8)
{
    DmaPlan p;
    p.bn = Nout % 128 == 0 ? 128 : 64;
    p.two_pass = q8 && Kred <= kTwoPassMaxKred;
    p.bm = (p.two_pass || Mrows < 256) ? 128 : ISEG_IGEMM_BM;
    p.splits = 1;
    if (q8 && !p.two_pass) {
        const int64_t blocks = ceil_div64(Mrows, p.bm) * (Nout / p.bn);
        const int nk = Kred / BK;
        while (p.splits < kMaxSplits && blocks * p.splits < ISEG_IGEMM_SPLIT_BLOCKS && nk / (2 * p.splits) >= 32)
            p.splits *= 2;
        // a short reduction that leaves the chip under one block per CU takes
        // 64-column tiles instead (twice the blocks); long reductions split
        // instead, where 128 x 128 tiles keep their higher MFMA rate
        if (p.splits == 1 && p.bn == 128 && blocks < 256) p.bn = 64;
    }
    return p;
}
// int32 workspace of a plan beyond the int16 staging: split partials
size_t dma_split_bytes(const DmaPlan& p, int64_t Mrows, int32_t Nout)
{
    return p.splits > 1 ? align256((size_t)p.splits * (size_t)Mrows * (size_t)Nout * 4) : 0;
}

// persistent short-reduction launch: as many tiles per block as leave about
// one round of blocks at the occupancy the LDS allows
#ifndef ISEG_CONV_SHORT
#define ISEG_CONV_SHORT 1
#endif
#ifndef ISEG_SHORT_TPB
#define ISEG_SHORT_TPB 0         // row tiles per block of the short kernel (0: sized from occupancy)
#endif
template <int MODE, int BN, int EPI>
int launch_short_t(const IgemmArgs& a, hipStream_t s, int64_t* nblk)
{
    const int kid = MODE == MODE_FWD ? ISEG_KID_CONV_FWD : ISEG_KID_CONV_BWD_DATA;
    const int nk = a.Kred / BK;
    const size_t lds = short_lds_bytes<BN, EPI>(nk);
    const int64_t nt = ceil_div64(a.Mrows, 128), ncol = a.Nout / BN;
    int64_t occ = (int64_t)((160 * 1024) / lds);
    occ = occ < 1 ? 1 : (occ > 4 ? 4 : occ);
    int64_t tpb = ISEG_SHORT_TPB > 0 ? ISEG_SHORT_TPB : ceil_div64(nt * ncol, 256 * occ);
    tpb = tpb < 1 ? 1 : tpb;
    dim3 grid((unsigned)ceil_div64(nt, tpb), (unsigned)ncol);
    if (lds > 65536 && !lds_limit((const void*)k_conv_short<MODE, BN, EPI>, lds)) return ISEG_ERR_DEVICE;
    ISEG_TIMED_LAUNCH(kid, s, (k_conv_short<MODE, BN, EPI>), grid, dim3(256), lds, s, a, (int)tpb);
    *nblk = (int64_t)grid.x * grid.y;
    return launch_ok();
}

// the register GEMM for 1x1 stride-1 convs (rows are contiguous pixels): each
// wave loads its own W fragments, so it pays off for few channel groups, at
// most two reduction steps and many pixels (measured on the DeepLabv3 shapes)
bool gemm_short_ok(const IgemmArgs& a)
{
    return ISEG_CONV_SHORT && a.R == 1 && a.S == 1 && a.sh == 1 && a.sw == 1 && a.ph == 0 && a.pw == 0 &&
           a.Ho == a.Hs && a.Wo == a.Ws && a.Kred % 64 == 0 && a.Kred <= 128 && a.Nout % 64 == 0 &&
           a.Nout <= 256 && a.Mrows >= 32768 &&
           (((uintptr_t)a.src | (uintptr_t)a.wmat) & 15) == 0 && ((uintptr_t)a.out8 & 3) == 0;
}

// the persistent LDS kernel: its double-buffered A tiles cost occupancy at
// three or four reduction steps, and it needs enough row tiles to fill the chip
bool lds_short_ok(const IgemmArgs& a) { return ISEG_CONV_SHORT && a.Kred <= 2 * BK && a.Mrows >= 16384; }

template <int MODE, int NK, int EPI>
int launch_gemm_short_t(const IgemmArgs& a, hipStream_t s, int64_t* nblk)
{
    const int kid = MODE == MODE_FWD ? ISEG_KID_CONV_FWD : ISEG_KID_CONV_BWD_DATA;
    constexpr int PB = NK <= 2 ? 32 : 16;
    const int64_t ncg = a.Nout / 64;
    const int64_t units = ceil_div64(a.Mrows, PB) * ncg;
    // waves: at most the units, at most 4 per SIMD over the chip, a multiple of
    // max(4, ncg) so that every wave keeps one channel group
    const int64_t q = ncg > 4 ? ncg : 4;
    int64_t waves = units < 4096 ? units : 4096;
    waves = ceil_div64(waves, q) * q;
    dim3 grid((unsigned)(waves / 4));
    ISEG_TIMED_LAUNCH(kid, s, (k_gemm_short<NK, EPI>), grid, dim3(256), 0, s, a);
    *nblk = grid.x;
    return launch_ok();
}

template <int MODE, int NK>
int launch_gemm_short_k(const IgemmArgs& a, int epi, hipStream_t s, int64_t* nblk)
{
    return epi == EPI_MAX ? launch_gemm_short_t<MODE, NK, EPI_MAX>(a, s, nblk)
                          : launch_gemm_short_t<MODE, NK, EPI_Q8>(a, s, nblk);
}

template <int MODE>
int launch_gemm_short(const IgemmArgs& a, int epi, hipStream_t s, int64_t* nblk)
{
    switch (a.Kred / 64) {
    case 1: return launch_gemm_short_k<MODE, 1>(a, epi, s, nblk);
    case 2: return launch_gemm_short_k<MODE, 2>(a, epi, s, nblk);
    case 3: return launch_gemm_short_k<MODE, 3>(a, epi, s, nblk);
    default: return launch_gemm_short_k<MODE, 4>(a, epi, s, nblk);
    }
}

template <int MODE>
int launch_short(const IgemmArgs& a, int epi, hipStream_t s, int64_t* nblk)
{
    if (gemm_short_ok(a)) return launch_gemm_short<MODE>(a, epi, s, nblk);
    if (a.Nout % 128 == 0)
        return epi == EPI_MAX ? launch_short_t<MODE, 128, EPI_MAX>(a, s, nblk)
                              : launch_short_t<MODE, 128, EPI_Q8>(a, s, nblk);
    return epi == EPI_MAX ? launch_short_t<MODE, 64, EPI_MAX>(a, s, nblk)
                          : launch_short_t<MODE, 64, EPI_Q8>(a, s, nblk);
}

template <int MODE, int BM, int BN, int EPI>
int launch_dma_t(const IgemmArgs& a, int splits, hipStream_t s, int64_t* nblk)
{
    const int kid = MODE == MODE_FWD ? ISEG_KID_CONV_FWD : ISEG_KID_CONV_BWD_DATA;
    dim3 grid((unsigned)ceil_div64(a.Mrows, BM), (unsigned)(a.Nout / BN), (unsigned)splits);
    size_t lds = (size_t)kStages * (BM + BN) * 64;
    const size_t epi_lds = EPI == EPI_STAGE16 ? (size_t)BM * (BN + 8) * 2 : EPI == EPI_Q8 ? (size_t)BM * (BN + 16) : 0;
    lds = lds > epi_lds ? lds : epi_lds;
    constexpr bool pipe = ISEG_IGEMM_PIPE != 0;
    if (lds > 65536 && !lds_limit((const void*)k_conv_igemm_dma<MODE, BM, BN, EPI, pipe>, lds))
        return ISEG_ERR_DEVICE;
    ISEG_TIMED_LAUNCH(kid, s, (k_conv_igemm_dma<MODE, BM, BN, EPI, pipe>), grid, dim3(256), lds, s, a);
    *nblk = (int64_t)grid.x * grid.y;
    return launch_ok();
}

template <int MODE, int BM, int BN>
int launch_dma_e(const IgemmArgs& a, int epi, int splits, hipStream_t s, int64_t* nblk)
{
    switch (epi) {
    case EPI_STAGE16: return launch_dma_t<MODE, BM, BN, EPI_STAGE16>(a, splits, s, nblk);
    case EPI_MAX: return launch_dma_t<MODE, BM, BN, EPI_MAX>(a, splits, s, nblk);
    case EPI_Q8: return launch_dma_t<MODE, BM, BN, EPI_Q8>(a, splits, s, nblk);
    case EPI_PART: return launch_dma_t<MODE, BM, BN, EPI_PART>(a, splits, s, nblk);
    default: return launch_dma_t<MODE, BM, BN, EPI_RAW>(a, splits, s, nblk);
    }
}

template <int MODE>
int launch_igemm_dma(const IgemmArgs& a, const DmaPlan& p, int epi, hipStream_t s, int64_t* nblk)
{
    if (p.bm == 256)
        return p.bn == 128 ? launch_dma_e<MODE, 256, 128>(a, epi, p.splits, s, nblk)
                           : launch_dma_e<MODE, 256, 64>(a, epi, p.splits, s, nblk);
    return p.bn == 128 ? launch_dma_e<MODE, 128, 128>(a, epi, p.splits, s, nblk)
                       : launch_dma_e<MODE, 128, 64>(a, epi, p.splits, s, nblk);
}

// sum of the split partials [splits][n] into out (in place allowed), with
// per-block max |sum| partials; four 16-byte groups per thread in flight
__global__ __launch_bounds__(256) void k_splitk_reduce(const int32_t* part, int32_t splits, int64_t n,
                                                       int32_t* out, uint64_t* pmax)
{
    constexpr int U = 4;
    uint32_t mx = 0;
    const int64_t n4 = n >> 2;
    const int64_t stride = (int64_t)gridDim.x * 256;
    for (int64_t i0 = (int64_t)blockIdx.x * 256 + threadIdx.x; i0 < n4; i0 += stride * U) {
        int4 v[U];
#pragma unroll
        for (int u = 0; u < U; u++) {
            const int64_t i = i0 + u * stride;
            v[u] = i < n4 ? ((const int4*)part)[i] : make_int4(0, 0, 0, 0);
        }
        for (int z = 1; z < splits; z++) {
            int4 w[U];
#pragma unroll
            for (int u = 0; u < U; u++) {
                const int64_t i = i0 + u * stride;
                w[u] = i < n4 ? ((const int4*)(part + (int64_t)z * n))[i] : make_int4(0, 0, 0, 0);
            }
#pragma unroll
            for (int u = 0; u < U; u++) { v[u].x += w[u].x; v[u].y += w[u].y; v[u].z += w[u].z; v[u].w += w[u].w; }
        }
#pragma unroll
        for (int u = 0; u < U; u++) {
            const int64_t i = i0 + u * stride;
            if (i < n4) {
                ((int4*)out)[i] = v[u];
                const uint32_t m01 = max((uint32_t)abs(v[u].x), (uint32_t)abs(v[u].y));
                const uint32_t m23 = max((uint32_t)abs(v[u].z), (uint32_t)abs(v[u].w));
                mx = max(mx, max(m01, m23));
            }
        }
    }
    if (pmax) block_store_max_u64(mx, pmax);
}

// int32 sums (+ per-block max partials) of any shape through the generic or
// tap kernels (the direct-to-LDS kernel is driven by igemm_dma_run)
template <int MODE>
int launch_igemm(const IgemmArgs& a, hipStream_t s, int64_t* nblk)
{
    *nblk = 0;
    if (a.Mrows > 0 && a.Nout > 0 && a.Ci % 64 == 0 &&
        (((uintptr_t)a.src | (uintptr_t)a.wmat) & 15) == 0) {
        const int kid = MODE == MODE_FWD ? ISEG_KID_CONV_FWD : ISEG_KID_CONV_BWD_DATA;
        unsigned gx = (unsigned)ceil_div64(a.Mrows, 128);
        if (a.Nout > 64) {
            dim3 grid(gx, (unsigned)ceil_div64(a.Nout, 128));
            ISEG_TIMED_LAUNCH(kid, s, (k_conv_igemm_tap<MODE, 128, 128>), grid, dim3(256), 0, s, a);
            *nblk = (int64_t)grid.x * grid.y;
        } else {
            ISEG_TIMED_LAUNCH(kid, s, (k_conv_igemm_tap<MODE, 128, 64>), dim3(gx, 1), dim3(256), 0, s, a);
            *nblk = gx;
        }
        return launch_ok();
    }
    return launch_igemm_generic<MODE>(a, s, nblk);
}

__global__ void k_exp_sum(int32_t* out, const int32_t* a, const int32_t* b);

// The whole direct-to-LDS path of a forward / backward-data conv (igemm_dma_ok
// and a 16-byte aligned output): raw sums, or final codes by two passes,
// split partials + reduce + requant, or int16 staging + requant.  `work` is
// the int32 / staging region of the workspace, `pmax` its max partials.
// true when every row tile of the plan skips at least one tap (the same test
// as the kernel's, over all tiles on the host)
template <int MODE>
bool every_tile_skips(const IgemmArgs& a, int bm)
{
    const int RS = a.R * a.S;
    if (!ISEG_IGEMM_TAPSKIP || RS == 1 || RS > 64 || a.sh != 1 || a.sw != 1) return false;
    const uint64_t all = RS == 64 ? ~0ull : (1ull << RS) - 1;
    const int64_t nt = ceil_div64(a.Mrows, bm);
    if (nt > 65536) return false;
    for (int64_t t = 0; t < nt; t++) {
        const int64_t m0 = t * bm, vr = a.Mrows - m0;
        if (live_taps<MODE>(a, m0, vr < bm ? (int)vr : bm) == all) return false;
    }
    return true;
}

template <int MODE>
int igemm_dma_run(IgemmArgs a, int out_mode, const int32_t* exp_a, const int32_t* exp_b, void* y,
                  int32_t* y_exp, uint64_t* pmax, int32_t* work, hipStream_t s)
{
    const DmaPlan p = dma_plan(a.Mrows, a.Nout, a.Kred, out_mode == ISEG_OUT_Q8);
    a.tap_balance = every_tile_skips<MODE>(a, p.bm) ? 1 : 0;
    int rc;
    int64_t nblk = 0;
    a.out16 = nullptr;
    a.tshift = nullptr;
    if (out_mode == ISEG_OUT_RAW) {
        conv_plan_set("dma");
        a.out = (int32_t*)y;
        a.pmax = nullptr;
        if ((rc = launch_igemm_dma<MODE>(a, p, EPI_RAW, s, &nblk))) return rc;
        hipLaunchKernelGGL(k_exp_sum, dim3(1), dim3(1), 0, s, y_exp, exp_a, exp_b);
        return launch_ok();
    }
    if (p.two_pass) {
        a.pmax = pmax;
        a.out8 = (int8_t*)y; a.exp_a = exp_a; a.exp_b = exp_b; a.out_exp = y_exp;   // both passes pick one kernel
        const bool sh = gemm_short_ok(a) || lds_short_ok(a);
        conv_plan_set(gemm_short_ok(a) ? "gemm_short" : sh ? "conv_short" : "dma_two_pass");
        if ((rc = sh ? launch_short<MODE>(a, EPI_MAX, s, &nblk) : launch_igemm_dma<MODE>(a, p, EPI_MAX, s, &nblk)))
            return rc;
        a.npmax = nblk;
        return sh ? launch_short<MODE>(a, EPI_Q8, s, &nblk) : launch_igemm_dma<MODE>(a, p, EPI_Q8, s, &nblk);
    }
    const int64_t n = a.Mrows * a.Nout;
    if (p.splits > 1) {
        conv_plan_set("dma_split");
        a.out = work;
        a.pmax = nullptr;
        if ((rc = launch_igemm_dma<MODE>(a, p, EPI_PART, s, &nblk))) return rc;
        // as many reduce blocks as the max-partial region holds for 128 x 64 tiles
        const int64_t cap = ceil_div64(a.Mrows, 128) * ceil_div64(a.Nout, 64);
        int64_t nb = ceil_div64(n / 4, 256 * 4);    // four 16-byte groups per thread
        nb = nb < cap ? nb : cap;
        nb = nb < 1 ? 1 : nb;
        hipLaunchKernelGGL(k_splitk_reduce, dim3((unsigned)nb), dim3(256), 0, s, work, (int32_t)p.splits, n, work,
                           pmax);
        if ((rc = launch_ok())) return rc;
        return launch_requant_apply(work, ISEG_I32, n, exp_a, exp_b, 0, 8, 0, 1, 0, 0, 0, ISEG_I8, y, y_exp,
                                    nullptr, s, pmax, nb);
    }
    conv_plan_set("dma_stage16");
    a.out16 = (int16_t*)work;
    a.tshift = (uint8_t*)work + align256((size_t)n * 2);
    a.pmax = pmax;
    if ((rc = launch_igemm_dma<MODE>(a, p, EPI_STAGE16, s, &nblk))) return rc;
    StageMap sm{p.bm, p.bn, 0, 0, 0, 0, 0, 0};
    return launch_requant_staged16(a.out16, a.tshift, a.Mrows, a.Nout, sm, exp_a, exp_b, 8, (int8_t*)y, y_exp,
                                   nullptr, s, pmax, nblk);
}

template <int MODE>
int launch_igemm_generic(const IgemmArgs& a, hipStream_t s, int64_t* nblk)
{
    *nblk = 0;
    if (a.Mrows <= 0 || a.Nout <= 0) return ISEG_OK;
    bool vec = (a.Ci % 16) == 0 && (((uintptr_t)a.src | (uintptr_t)a.wmat) & 15) == 0;
    dim3 block(256);
    unsigned gx = (unsigned)ceil_div64(a.Mrows, 128);
    const int kid = MODE == MODE_FWD ? ISEG_KID_CONV_FWD : ISEG_KID_CONV_BWD_DATA;
    if (a.Nout > 64) {
        dim3 grid(gx, (unsigned)ceil_div64(a.Nout, 128));
        if (vec) ISEG_TIMED_LAUNCH(kid, s, (k_conv_igemm<MODE, true, 128, 128>), grid, block, 0, s, a);
        else ISEG_TIMED_LAUNCH(kid, s, (k_conv_igemm<MODE, false, 128, 128>), grid, block, 0, s, a);
        *nblk = (int64_t)grid.x * grid.y;
    } else {
        dim3 grid(gx, 1);
        if (vec) ISEG_TIMED_LAUNCH(kid, s, (k_conv_igemm<MODE, true, 128, 64>), grid, block, 0, s, a);
        else ISEG_TIMED_LAUNCH(kid, s, (k_conv_igemm<MODE, false, 128, 64>), grid, block, 0, s, a);
        *nblk = gx;
    }
    return launch_ok();
}

// ---------------------------------------------------------------------------
// weights KRSC -> CRSK for the backward-data GEMM
// ---------------------------------------------------------------------------
// One 64 x 64 tile of a weight transpose: w[K][RS][C] -> wt[C][RS][K] (tap
// rs of the source goes to tap RS-1-rs when `flip`, the backward-data filter
// of a stride-1 conv).  The tile (k0.., c0.., tap rs) is read as 64 rows of
// 64 contiguous channel bytes and written as 64 rows of 64 contiguous output
// channels through an LDS tile (one padding byte per row against bank
// conflicts); 256 threads, every index in 32-bit arithmetic.
__device__ __forceinline__ void wt_tile(const int8_t* __restrict__ w, int8_t* __restrict__ wt, int32_t K,
                                        int32_t RS, int32_t C, bool flip, int32_t k0, int32_t c0, int32_t rs)
{
    __shared__ int8_t t[64][65];
    const int rso = flip ? RS - 1 - rs : rs;
    if (((C | K) & 3) == 0 && ((((uintptr_t)w) | ((uintptr_t)wt)) & 3) == 0) {
        // dword loads and stores: four channels per lane in, four k per lane out
        const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
#pragma unroll
        for (int j = 0; j < 4; j++) {
            const int k = k0 + ty + 16 * j, c = c0 + 4 * tx;
            const uint32_t v = (k < K && c < C) ? *(const uint32_t*)(w + ((uint32_t)k * RS + rs) * (uint32_t)C + c) : 0u;
#pragma unroll
            for (int e = 0; e < 4; e++) t[ty + 16 * j][4 * tx + e] = (int8_t)(v >> (8 * e));
        }
        __syncthreads();
#pragma unroll
        for (int j = 0; j < 4; j++) {
            const int c = c0 + ty + 16 * j, k = k0 + 4 * tx;
            if (c < C && k < K) {
                uint32_t v = 0;
#pragma unroll
                for (int e = 0; e < 4; e++) v |= (uint32_t)(uint8_t)t[4 * tx + e][ty + 16 * j] << (8 * e);
                *(uint32_t*)(wt + ((uint32_t)c * RS + rso) * (uint32_t)K + k) = v;
            }
        }
        return;
    }
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
#pragma unroll
    for (int j = 0; j < 16; j++) {
        const int k = k0 + ty + 4 * j, c = c0 + tx;
        t[ty + 4 * j][tx] = (k < K && c < C) ? w[((uint32_t)k * RS + rs) * (uint32_t)C + c] : (int8_t)0;
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 16; j++) {
        const int c = c0 + ty + 4 * j, k = k0 + tx;
        if (c < C && k < K) wt[((uint32_t)c * RS + rso) * (uint32_t)K + k] = t[tx][ty + 4 * j];
    }
}

// grid (ceil(C/64), ceil(K/64), RS)
__global__ __launch_bounds__(256) void k_w_transpose_t(const int8_t* __restrict__ w, int8_t* __restrict__ wt,
                                                       int32_t K, int32_t RS, int32_t C, int32_t flip)
{
    wt_tile(w, wt, K, RS, C, flip != 0, blockIdx.y * 64, blockIdx.x * 64, blockIdx.z);
}

int launch_w_transpose(const int8_t* w, int8_t* wt, int64_t K, int64_t RS, int64_t C, bool flip, hipStream_t s)
{
    dim3 grid((unsigned)ceil_div64(C, 64), (unsigned)ceil_div64(K, 64), (unsigned)RS);
    hipLaunchKernelGGL(k_w_transpose_t, grid, dim3(256), 0, s, w, wt, (int32_t)K, (int32_t)RS, (int32_t)C,
                       (int32_t)flip);
    return launch_ok();
}

// every tensor of a descriptor table in one launch: block b takes the tile
// b - tile_begin of the last descriptor whose tile_begin <= b
__global__ __launch_bounds__(256) void k_w_transpose_multi(const iseg_wt_desc* __restrict__ d, int32_t n)
{
    const int64_t b = blockIdx.x;
    int lo = 0, hi = n - 1;
    while (lo < hi) {                       // last descriptor with tile_begin <= b
        const int mid = (lo + hi + 1) >> 1;
        if (d[mid].tile_begin <= b) lo = mid; else hi = mid - 1;
    }
    const iseg_wt_desc e = d[lo];
    const int32_t tc = (e.C + 63) / 64, tk = (e.K + 63) / 64;
    const int64_t t = b - e.tile_begin;
    const int32_t rs = (int32_t)(t / ((int64_t)tc * tk));
    if (rs >= e.RS) return;                 // total_tiles larger than the table's sum
    const int32_t r2 = (int32_t)(t - (int64_t)rs * tc * tk);
    wt_tile(e.w, e.wt, e.K, e.RS, e.C, e.kind == ISEG_WT_CRSK_FLIP, (r2 / tc) * 64, (r2 % tc) * 64, rs);
}

// channel padding for small C: out[pix][c] = c < C ? in[pix][c] : 0
__global__ void k_pad_channels(const int8_t* __restrict__ in, int8_t* __restrict__ out, int64_t npix,
                               int32_t C, int32_t Cp)
{
    int64_t n = npix * Cp;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        int64_t pix = i / Cp;
        int32_t c = (int32_t)(i - pix * Cp);
        out[i] = c < C ? in[pix * C + c] : (int8_t)0;
    }
}

// drop the padded channels of int64 weight-gradient sums
__global__ void k_unpad_i64(const long long* __restrict__ in, long long* __restrict__ out, int64_t rows,
                            int32_t C, int32_t Cp)
{
    int64_t n = rows * C;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        int64_t r = i / C;
        out[i] = in[r * Cp + (i - r * C)];
    }
}

static int64_t padded_c(int64_t C) { return (C % 16 == 0 || C > 64) ? C : ((C + 15) / 16) * 16; }

static int launch_pad(const int8_t* in, int8_t* out, int64_t npix, int64_t C, int64_t Cp, hipStream_t s)
{
    if (npix <= 0) return ISEG_OK;
    hipLaunchKernelGGL(k_pad_channels, dim3(grid_for(npix * Cp, 256, 8192)), dim3(256), 0, s, in, out,
                       npix, (int32_t)C, (int32_t)Cp);
    return launch_ok();
}

// A 1x1 stride-1 conv whose reduction channels for backward-data (its K,
// e.g. a classifier's class count) are not a multiple of 64: dy and the
// transposed weights padded with zero channels to the next multiple of 64 take
// the direct-to-LDS path (the zero channels add nothing to the sums).
static int64_t kpad_to(int64_t K) { return ceil_div64(K, 64) * 64; }

static bool kpad_ok(const iseg_conv_geom* g)
{
    return g->R == 1 && g->S == 1 && g->stride_h == 1 && g->stride_w == 1 && g->pad_h == 0 && g->pad_w == 0 &&
           g->K % 64 != 0 && g->C % 64 == 0 && g->N > 0 && g->N * g->H * g->W < ((int64_t)1 << 31);
}

static size_t kpad_bytes(const iseg_conv_geom* g)
{
    if (!kpad_ok(g)) return 0;
    const int64_t Kp = kpad_to(g->K);
    return align256((size_t)(g->N * g->H * g->W * Kp)) + align256((size_t)(g->C * Kp));
}

// wt[c][k] = w[k][c] for k < K, 0 up to Kp (1x1 weights KC -> C x Kp)
__global__ void k_wt_pad_1x1(const int8_t* __restrict__ w, int8_t* __restrict__ wt, int32_t K, int32_t C, int32_t Kp)
{
    const int64_t n = (int64_t)C * Kp;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        const int32_t c = (int32_t)(i / Kp), k = (int32_t)(i - (int64_t)c * Kp);
        wt[i] = k < K ? w[(int64_t)k * C + c] : (int8_t)0;
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
    int32_t* part;           // or, when set: int32 [split][K][RSC], stored (k_conv_wgrad_tr)
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

int launch_wgrad_generic(WgradArgs a, hipStream_t s);

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

// Backward-weight when C % 64 == 0: a block owns one filter tap (r,s), a
// 64-channel chunk of C and BM output channels, so every column of its tile
// shares the tap.  Per 64-pixel step, 64 lanes turn the pixel indices into
// source offsets once (staged in LDS); the dy and x tiles are then plain
// dword gathers, transposed 4x4 in registers into pixel-contiguous LDS rows.
template <int BM>
__global__ __launch_bounds__(256) void k_conv_wgrad_tap(WgradArgs a)
{
    constexpr int BN = 64;
    constexpr int WM = BM / 2, WN = BN / 2;
    constexpr int TM = WM / 16, TN = WN / 16;
    constexpr int QA = BM / 64;
    __shared__ __attribute__((aligned(16))) int8_t As[BM * ROW];
    __shared__ __attribute__((aligned(16))) int8_t Bs[BN * ROW];
    __shared__ int64_t soff[BK];

    const int tid = threadIdx.x;
    const int nch = a.C / BN;
    const int tap = blockIdx.x / nch;
    const int c0 = (blockIdx.x - tap * nch) * BN;
    const int r = tap / a.S, s = tap - (tap / a.S) * a.S;
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
        if (tid < BK) {
            int64_t pix = pb + tid;
            int64_t off = -1;
            if (pix < pend) {
                int32_t n = (int32_t)(pix / PQ);
                int32_t rem = (int32_t)(pix - (int64_t)n * PQ);
                int32_t p = rem / a.Q, q = rem - (rem / a.Q) * a.Q;
                int ih = p * a.sh - a.ph + r * a.dh, iw = q * a.sw - a.pw + s * a.dw;
                if (ih >= 0 && iw >= 0 && ih < a.H && iw < a.W)
                    off = (((int64_t)n * a.H + ih) * a.W + iw) * a.C + c0;
            }
            soff[tid] = off;
        }
        __syncthreads();
        uint32_t ta[QA][4], tb[4];
#pragma unroll
        for (int qq = 0; qq < QA; qq++) {
            int bi = tid + 256 * qq;
            int cg = bi % (BM / 4), pg = bi / (BM / 4);
            int kc = k0 + cg * 4;
            uint32_t in[4];
#pragma unroll
            for (int i = 0; i < 4; i++) {
                int64_t pix = pb + pg * 4 + i;
                in[i] = (pix < pend && kc < a.K) ? *(const uint32_t*)(a.dy + pix * a.K + kc) : 0u;
            }
            transpose4x4(in, ta[qq]);
        }
        {
            int cg = tid % (BN / 4), pg = tid / (BN / 4);
            uint32_t in[4];
#pragma unroll
            for (int i = 0; i < 4; i++) {
                int64_t off = soff[pg * 4 + i];
                in[i] = off >= 0 ? *(const uint32_t*)(a.x + off + cg * 4) : 0u;
            }
            transpose4x4(in, tb);
        }
#pragma unroll
        for (int qq = 0; qq < QA; qq++) {
            int bi = tid + 256 * qq;
            int cg = bi % (BM / 4), pg = bi / (BM / 4);
#pragma unroll
            for (int c = 0; c < 4; c++) *(uint32_t*)&As[(cg * 4 + c) * ROW + pg * 4] = ta[qq][c];
        }
        {
            int cg = tid % (BN / 4), pg = tid / (BN / 4);
#pragma unroll
            for (int c = 0; c < 4; c++) *(uint32_t*)&Bs[(cg * 4 + c) * ROW + pg * 4] = tb[c];
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

    const int colbase = tap * a.C + c0;
#pragma unroll
    for (int i = 0; i < TM; i++)
#pragma unroll
        for (int j = 0; j < TN; j++) {
            int col = colbase + wn * WN + j * 16 + lrow;
#pragma unroll
            for (int e = 0; e < 4; e++) {
                int k = k0 + wm * WM + i * 16 + (lane >> 4) * 4 + e;
                int32_t v = acc[i][j][e];
                if (k >= a.K) continue;
                if (a.part)
                    a.part[((int64_t)blockIdx.z * a.K + k) * a.RSC + col] = v;
                else if (v != 0)
                    atomicAdd(&a.acc[(int64_t)k * a.RSC + col], (unsigned long long)(int64_t)v);
            }
        }
}

// Backward-weight with transposing LDS reads (C % 64 == 0, K % 16 == 0).
// Tiles are staged in their natural layout -- [pixel][channel] rows of dy and
// of the tap-shifted x -- with plain 16-byte copies, and the MFMA operands
// (16 consecutive pixels of one channel per lane) come out of ds_read_b64_tr_b8:
// within a 16-lane group, output lane j's byte i is byte (j mod 8) of source
// lane 2i + j/8, so source lane 2i + h pointing at (pixel i, channels c0 + 8h)
// hands lane j channel c0 + j of pixels 0..7.  A block owns BM output
// channels, TAPS filter taps and one 64-channel chunk of C.
typedef int v2i_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ v4i tr8_frag(const int8_t* lds_rows, int row_bytes, int col0, int lane)
{
    // 16-lane group g = lane/16 covers pixels 16g .. 16g+15 of the tile
    const int g = lane >> 4, sl = lane & 15;
    const int i = sl >> 1, h = sl & 1;
    const int8_t* p0 = lds_rows + (16 * g + i) * row_bytes + col0 + 8 * h;
    const int8_t* p1 = p0 + 8 * row_bytes;
    v2i_t a = __builtin_amdgcn_ds_read_tr8_b64_v2i32((__attribute__((address_space(3))) v2i_t*)p0);
    v2i_t b = __builtin_amdgcn_ds_read_tr8_b64_v2i32((__attribute__((address_space(3))) v2i_t*)p1);
    return (v4i){a.x, a.y, b.x, b.y};
}

template <int BM, int TAPS>
__global__ __launch_bounds__(256) void k_conv_wgrad_tr(WgradArgs a)
{
    constexpr int BN = 64 * TAPS;
    constexpr int RA = BM + 16;               // LDS row bytes of the dy tile
    constexpr int RB = 80;                    // LDS row bytes of an x tile (64 channels)
    constexpr int WM = BM / 2, WN = BN / 2;
    constexpr int TM = WM / 16, TN = WN / 16;
    constexpr int PA = BM / 64;               // 16-byte dy pieces per thread
    constexpr int D = 4;                      // steps of global loads in flight
    __shared__ __attribute__((aligned(16))) int8_t As[2][BK * RA];
    __shared__ __attribute__((aligned(16))) int8_t Bs[2][TAPS][BK * RB];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int nch = a.C / 64;
    const int tg = blockIdx.x / nch;
    const int c0 = (blockIdx.x - tg * nch) * 64;
    const int k0 = blockIdx.y * BM;
    // 32-bit offsets: x and dy are below 2^31 bytes (wgrad_tr_ok)
    const int32_t pbeg = (int32_t)(blockIdx.z * a.pix_per_split);
    const int32_t pend = (int32_t)(pbeg + a.pix_per_split < a.NPQ ? pbeg + a.pix_per_split : a.NPQ);

    // this thread stages pixel (step base + tid/4), 16-byte part tid%4
    const int prow = tid >> 2, part = tid & 3;
    int dr[TAPS], ds[TAPS];                   // input pixel (p sh + dr, q sw + ds) of output pixel (p, q)
    bool tok[TAPS];
#pragma unroll
    for (int t = 0; t < TAPS; t++) {
        int tap = tg * TAPS + t;
        tok[t] = tap < a.R * a.S;
        const int tr = tok[t] ? tap / a.S : 0;
        dr[t] = tr * a.dh - a.ph;
        ds[t] = (tok[t] ? tap - tr * a.S : 0) * a.dw - a.pw;
    }
    // load cursor: coordinates of this thread's pixel, advanced 64 pixels (dp
    // rows and dq columns) per step
    int32_t pix = pbeg + prow;
    const int32_t PQ = a.P * a.Q;
    int32_t pn = pix / PQ;
    int32_t rem = pix - pn * PQ;
    int32_t pp = rem / a.Q, pq = rem - (rem / a.Q) * a.Q;
    const int32_t dp = BK / a.Q, dq = BK - (BK / a.Q) * a.Q;
    const uint32_t HWC = (uint32_t)a.H * a.W * a.C, WC = (uint32_t)a.W * a.C;

    int4 ra[D][PA], rb[D][TAPS];
    auto load = [&](int4* pa, int4* pb) {
        const bool ok = pix < pend;
#pragma unroll
        for (int j = 0; j < PA; j++) {          // k0 + part * 16 + 64 j < K: K % BM == 0
            const uint32_t off = (uint32_t)pix * (uint32_t)a.K + (uint32_t)(k0 + part * 16 + 64 * j);
            pa[j] = ok ? *(const int4*)(a.dy + off) : make_int4(0, 0, 0, 0);
        }
#pragma unroll
        for (int t = 0; t < TAPS; t++) {
            const int ih = pp * a.sh + dr[t], iw = pq * a.sw + ds[t];
            const bool v = ok && tok[t] && (uint32_t)ih < (uint32_t)a.H && (uint32_t)iw < (uint32_t)a.W;
            // unsigned (wrapping) arithmetic: an offset out of range is never loaded
            const uint32_t off = (uint32_t)pn * HWC + (uint32_t)ih * WC + (uint32_t)iw * (uint32_t)a.C +
                                 (uint32_t)(c0 + part * 16);
            pb[t] = v ? *(const int4*)(a.x + off) : make_int4(0, 0, 0, 0);
        }
        pix += BK;
        pq += dq;
        pp += dp;
        if (pq >= a.Q) { pq -= a.Q; ++pp; }
        while (pp >= a.P) { pp -= a.P; ++pn; }
    };
    auto store = [&](int buf, const int4* pa, const int4* pb) {
#pragma unroll
        for (int j = 0; j < PA; j++) *(int4*)&As[buf][prow * RA + part * 16 + 64 * j] = pa[j];
#pragma unroll
        for (int t = 0; t < TAPS; t++) *(int4*)&Bs[buf][t][prow * RB + part * 16] = pb[t];
    };

    v4i acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; i++)
#pragma unroll
        for (int j = 0; j < TN; j++) acc[i][j] = (v4i){0, 0, 0, 0};

    const int nsteps = (int)((pend - pbeg + BK - 1) / BK);
#pragma unroll
    for (int u = 0; u < D; u++)
        if (u < nsteps) load(ra[u], rb[u]);
    store(0, ra[0], rb[0]);
    __syncthreads();
    for (int st0 = 0; st0 < nsteps; st0 += D) {
#pragma unroll
        for (int u = 0; u < D; u++) {
            const int st = st0 + u;
            if (st < nsteps) {
                const int8_t* A = As[st & 1];
                v4i fa[TM], fb[TN];
#pragma unroll
                for (int i = 0; i < TM; i++) fa[i] = tr8_frag(A, RA, wm * WM + i * 16, lane);
#pragma unroll
                for (int j = 0; j < TN; j++) {
                    const int col = wn * WN + j * 16;
                    fb[j] = tr8_frag(Bs[st & 1][col >> 6], RB, col & 63, lane);
                }
#pragma unroll
                for (int i = 0; i < TM; i++)
#pragma unroll
                    for (int j = 0; j < TN; j++)
                        acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[i], fb[j], acc[i][j], 0, 0, 0);
                // stage the next step (its loads were issued D-1 steps ago), then
                // reuse this slot of the ring for step st + D
                if (st + 1 < nsteps) store((st + 1) & 1, ra[(u + 1) % D], rb[(u + 1) % D]);
                if (st + D < nsteps) load(ra[u], rb[u]);
                __syncthreads();
            }
        }
    }

#pragma unroll
    for (int i = 0; i < TM; i++)
#pragma unroll
        for (int j = 0; j < TN; j++) {
            const int colt = wn * WN + j * 16 + (lane & 15);
            const int t = colt >> 6;
            const int tap = tg * TAPS + t;
            if (tap >= a.R * a.S) continue;
            const int64_t col = (int64_t)tap * a.C + c0 + (colt & 63);
#pragma unroll
            for (int e = 0; e < 4; e++) {
                int k = k0 + wm * WM + i * 16 + (lane >> 4) * 4 + e;
                int32_t v = acc[i][j][e];
                if (k >= a.K) continue;
                if (a.part)
                    a.part[((int64_t)blockIdx.z * a.K + k) * a.RSC + col] = v;
                else if (v != 0)
                    atomicAdd(&a.acc[(int64_t)k * a.RSC + col], (unsigned long long)(int64_t)v);
            }
        }
}

// Backward-weight, all taps in one block (C % 64 == 0, K % 64 == 0, R*S = 9):
// wave w owns filter tap w, the block owns 64 output channels (k), one
// 64-channel chunk of C and a run of output pixels, and writes its exact
// int32 partial tile (no atomics; k_wgrad_reduce adds the splits in int64).
// Per step (64 output pixels) an LDS stage holds the dy tile (64 pixel rows
// of 64 output channels), shared by every wave, and one x tile per tap (64
// rows of 64 input channels, the tap's shifted pixels; zeros come from a zero
// page for padding and past the split).  The stages are filled by
// direct-to-LDS loads (global_load_lds, 16 bytes per lane) in a ring of
// kWgStages (four stages of 40 KB: the whole LDS), so loads run three steps
// ahead without holding registers; waves 0-3 also load the dy rows, so the
// wait counts differ by wave.  Rows are 64 bytes, unpadded; the 16-byte part
// p of row R sits at part p ^ f(R), f(R) = ((R >> 1) ^ (R >> 4)) & 3, so the
// transposing reads (rows 16 g + i, i < 8, of four lane groups g) spread
// over the banks two rows per bank.
constexpr int kWgStages = 4;

__device__ __forceinline__ int wg_sw(int row) { return ((row >> 1) ^ (row >> 4)) & 3; }

// The four 16 x 64 fragments of a tile (columns 0, 16, 32, 48), read with
// ds_read_b64_tr_b8 in one asm block that ends in its own lgkmcnt wait: the
// compiler's form of that read carries no LDS alias information, so after
// direct-to-LDS loads it would wait for every one in flight (vmcnt 0) before
// the read, and the ring would no longer run ahead.
__device__ __forceinline__ uint32_t lds_off(const int8_t* p)
{
    return (uint32_t)(size_t)(const __attribute__((address_space(3))) int8_t*)p;
}

__device__ __forceinline__ void tr8_frags_sw(const int8_t* tile, int lane, v4i* f)
{
    const int g = lane >> 4, sl = lane & 15;
    const int i = sl >> 1, h = sl & 1;
    const int r0 = 16 * g + i, r1 = r0 + 8;
    uint32_t ad[8];
#pragma unroll
    for (int c = 0; c < 4; c++) {
        ad[2 * c] = lds_off(tile + r0 * 64 + ((c ^ wg_sw(r0)) << 4) + 8 * h);
        ad[2 * c + 1] = lds_off(tile + r1 * 64 + ((c ^ wg_sw(r1)) << 4) + 8 * h);
    }
    v2i_t v0, v1, v2, v3, v4, v5, v6, v7;
    asm volatile("ds_read_b64_tr_b8 %0, %8\n\t"
                 "ds_read_b64_tr_b8 %1, %9\n\t"
                 "ds_read_b64_tr_b8 %2, %10\n\t"
                 "ds_read_b64_tr_b8 %3, %11\n\t"
                 "ds_read_b64_tr_b8 %4, %12\n\t"
                 "ds_read_b64_tr_b8 %5, %13\n\t"
                 "ds_read_b64_tr_b8 %6, %14\n\t"
                 "ds_read_b64_tr_b8 %7, %15\n\t"
                 "s_waitcnt lgkmcnt(0)"
                 : "=&v"(v0), "=&v"(v1), "=&v"(v2), "=&v"(v3), "=&v"(v4), "=&v"(v5), "=&v"(v6), "=&v"(v7)
                 : "v"(ad[0]), "v"(ad[1]), "v"(ad[2]), "v"(ad[3]), "v"(ad[4]), "v"(ad[5]), "v"(ad[6]), "v"(ad[7])
                 : "memory");
    f[0] = (v4i){v0.x, v0.y, v1.x, v1.y};
    f[1] = (v4i){v2.x, v2.y, v3.x, v3.y};
    f[2] = (v4i){v4.x, v4.y, v5.x, v5.y};
    f[3] = (v4i){v6.x, v6.y, v7.x, v7.y};
}

size_t wgrad_taps_lds(int RS) { return (size_t)kWgStages * (1 + RS) * BK * 64; }

template <int RS>
__global__ __launch_bounds__(64 * RS) void k_conv_wgrad_taps(WgradArgs a, int32_t* __restrict__ part_out)
{
    constexpr int S = kWgStages;
    constexpr int TILE = BK * 64;                       // 64 rows of 64 bytes
    constexpr int STAGE = (1 + RS) * TILE;              // the dy tile, then one x tile per tap
    static_assert((S - 1) * 5 < 64, "vmcnt range");
    extern __shared__ __attribute__((aligned(16))) int8_t smem[];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;         // wave = tap
    const int nch = a.C / 64;
    const int c0 = (blockIdx.x % nch) * 64;
    const int k0 = (blockIdx.x / nch) * 64;
    // 32-bit offsets: x and dy are below 2^31 bytes (checked by the caller)
    const int32_t pbeg = (int32_t)(blockIdx.y * a.pix_per_split);
    const int32_t pend = (int32_t)(pbeg + a.pix_per_split < a.NPQ ? pbeg + a.pix_per_split : a.NPQ);
    const int32_t PQ = a.P * a.Q;
    const int wv = __builtin_amdgcn_readfirstlane(wave);            // uniform: LDS bases in scalar registers
    const int tr = wv / a.S, ts = wv - (wv / a.S) * a.S;
    const int rin = lane >> 2;                          // row of this lane in a 16-row load
    // the zero page's address held in scalar registers (not re-derived per load)
    uint64_t zbits = (uint64_t)(uintptr_t)g_conv_zero;
    asm volatile("" : "+s"(zbits));
    const int8_t* zp = (const int8_t*)(uintptr_t)zbits;
    // Cursor j (pixel 16 j + rin of the step being issued) carries its output
    // coordinates, the tap's input coordinates (ih, iw) = (p sh + r dh - ph,
    // q sw + s dw - pw) and the byte offset of that input pixel's 16-byte part
    // (unsigned, wrapping: meaningful only where (ih, iw) is in the image).
    // A step of 64 pixels advances dp rows and dq columns.
    const int32_t dp = BK / a.Q, dq = BK - (BK / a.Q) * a.Q;
    const uint32_t C = (uint32_t)a.C, WC = (uint32_t)a.W * C, HWC = (uint32_t)a.H * WC;
    const uint32_t o_q = (uint32_t)(dq * a.sw) * C + (uint32_t)(dp * a.sh) * WC;   // per step
    const uint32_t o_row = (uint32_t)a.sh * WC - (uint32_t)(a.Q * a.sw) * C;       // column wrap
    const uint32_t o_img = HWC - (uint32_t)(a.P * a.sh) * WC;                       // row wrap
    int32_t xpix[4], xp[4], xq[4], ih[4], iw[4];
    uint32_t xoff[4];
#pragma unroll
    for (int j = 0; j < 4; j++) {
        xpix[j] = pbeg + 16 * j + rin;
        const int32_t pp = xpix[j] < a.NPQ ? xpix[j] : 0;
        const int32_t n = pp / PQ, rem = pp - n * PQ;
        xp[j] = rem / a.Q;
        xq[j] = rem - xp[j] * a.Q;
        ih[j] = xp[j] * a.sh + tr * a.dh - a.ph;
        iw[j] = xq[j] * a.sw + ts * a.dw - a.pw;
        const int xpart = (lane & 3) ^ wg_sw(16 * j + rin);
        xoff[j] = (uint32_t)n * HWC + (uint32_t)ih[j] * WC + (uint32_t)iw[j] * C + (uint32_t)(c0 + xpart * 16);
    }
    const int dpart = (lane & 3) ^ wg_sw(16 * (wv & 3) + rin);
    uint32_t doff = (uint32_t)(pbeg + 16 * (wv & 3) + rin) * (uint32_t)a.K + (uint32_t)(k0 + dpart * 16);
    const uint32_t dstep = (uint32_t)BK * (uint32_t)a.K;
    const int nsteps = (pend - pbeg + BK - 1) / BK;

    auto issue = [&](int st) {
        if (st < nsteps) {
            int8_t* base = smem + (st % S) * STAGE;
#pragma unroll
            for (int j = 0; j < 4; j++) {
                const bool v = xpix[j] < pend && (uint32_t)ih[j] < (uint32_t)a.H && (uint32_t)iw[j] < (uint32_t)a.W;
                dma16(v ? a.x + xoff[j] : zp, base + (1 + wv) * TILE + j * 1024);
                xpix[j] += BK;
                xq[j] += dq;
                xp[j] += dp;
                ih[j] += dp * a.sh;
                iw[j] += dq * a.sw;
                xoff[j] += o_q;
                if (xq[j] >= a.Q) {
                    xq[j] -= a.Q; ++xp[j];
                    ih[j] += a.sh; iw[j] -= a.Q * a.sw;
                    xoff[j] += o_row;
                }
                while (xp[j] >= a.P) {
                    xp[j] -= a.P;
                    ih[j] -= a.P * a.sh;
                    xoff[j] += o_img;
                }
            }
            if (wv < 4) {
                const int32_t pix = pbeg + st * BK + 16 * wv + rin;
                dma16(pix < pend ? a.dy + doff : zp, base + wv * 1024);
                doff += dstep;
            }
        }
    };

    v4i acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; i++)
#pragma unroll
        for (int j = 0; j < 4; j++) acc[i][j] = (v4i){0, 0, 0, 0};

#pragma unroll
    for (int st = 0; st < S - 1; st++) issue(st);
    for (int st = 0; st < nsteps; st++) {
        // this wave's loads of step st have landed (those of the next S - 2
        // steps may still be in flight) and its reads of step st - 1 are done;
        // after the barrier every wave's are, so step st - 1's stage is free
        if (st + S - 2 >= nsteps) wait_vm_lgkm0<0>();       // the last steps: fewer loads behind
        else if (wv < 4) wait_vm_lgkm0<(S - 2) * 5>();      // x rows and a dy row per step
        else wait_vm_lgkm0<(S - 2) * 4>();                  // x rows only
        __builtin_amdgcn_s_barrier();
        issue(st + S - 1);
        const int8_t* A = smem + (st % S) * STAGE;
        const int8_t* B = A + (1 + wv) * TILE;
        v4i fa[4], fb[4];
        tr8_frags_sw(A, lane, fa);
        tr8_frags_sw(B, lane, fb);
#pragma unroll
        for (int i = 0; i < 4; i++)
#pragma unroll
            for (int j = 0; j < 4; j++)
                acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[i], fb[j], acc[i][j], 0, 0, 0);
    }
    wait_vm<0>();                                       // no load into LDS outlives the block

    // exact int32 partial tile of this split: part_out[split][k][tap * C + c]
    int32_t* outp = part_out + (int64_t)blockIdx.y * a.K * a.RSC;
#pragma unroll
    for (int i = 0; i < 4; i++)
#pragma unroll
        for (int j = 0; j < 4; j++) {
            const int64_t col = (int64_t)wave * a.C + c0 + j * 16 + (lane & 15);
#pragma unroll
            for (int e = 0; e < 4; e++) {
                const int k = k0 + i * 16 + (lane >> 4) * 4 + e;
                outp[(int64_t)k * a.RSC + col] = acc[i][j][e];
            }
        }
}

// Sum the per-split int32 partials in int64 (and take their max |.| for the
// quantizer).  A block owns 256 consecutive elements (one int4 per lane); its
// 8 waves take every 8th split, four loads in flight each, then fold in LDS.
constexpr int kRedWaves = 8;
__global__ __launch_bounds__(64 * kRedWaves) void k_wgrad_reduce(const int32_t* __restrict__ part, int64_t n,
                                                                 int splits, long long* __restrict__ out,
                                                                 uint64_t* pmax)
{
    __shared__ long long red[kRedWaves][256];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t e0 = (int64_t)blockIdx.x * 256 + lane * 4;
    long long s[4] = {0, 0, 0, 0};
    if (e0 < n) {                         // n % 4 == 0: K is a multiple of 64
        int k = wave;
        for (; k + 3 * kRedWaves < splits; k += 4 * kRedWaves) {
            int4 v[4];
#pragma unroll
            for (int u = 0; u < 4; u++) v[u] = *(const int4*)(part + (int64_t)(k + u * kRedWaves) * n + e0);
#pragma unroll
            for (int u = 0; u < 4; u++) { s[0] += v[u].x; s[1] += v[u].y; s[2] += v[u].z; s[3] += v[u].w; }
        }
        for (; k < splits; k += kRedWaves) {
            int4 v = *(const int4*)(part + (int64_t)k * n + e0);
            s[0] += v.x; s[1] += v.y; s[2] += v.z; s[3] += v.w;
        }
    }
#pragma unroll
    for (int u = 0; u < 4; u++) red[wave][lane * 4 + u] = s[u];
    __syncthreads();
    uint64_t mx = 0;
    if (threadIdx.x < 256) {
        const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
        long long t = 0;
#pragma unroll
        for (int w = 0; w < kRedWaves; w++) t += red[w][threadIdx.x];
        if (e < n) {
            out[e] = t;
            mx = t < 0 ? (uint64_t)(-t) : (uint64_t)t;
        }
    }
    if (pmax) block_store_max_u64(mx, pmax);
}

// Two-level variant for weight tensors too small to fill the chip with one
// block per 256 weights: blockIdx.y takes a chunk of the splits and writes an
// int64 partial; k_wgrad_reduce_fin adds the chunks in order.
__global__ __launch_bounds__(256) void k_wgrad_reduce_part(const int32_t* __restrict__ part, int64_t n,
                                                           int splits, int chunk, long long* __restrict__ out2)
{
    const int64_t e0 = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
    if (e0 >= n) return;                  // n % 4 == 0
    const int k0 = blockIdx.y * chunk;
    const int k1 = k0 + chunk < splits ? k0 + chunk : splits;
    long long s[4] = {0, 0, 0, 0};
    int k = k0;
    for (; k + 3 < k1; k += 4) {
        int4 v[4];
#pragma unroll
        for (int u = 0; u < 4; u++) v[u] = *(const int4*)(part + (int64_t)(k + u) * n + e0);
#pragma unroll
        for (int u = 0; u < 4; u++) { s[0] += v[u].x; s[1] += v[u].y; s[2] += v[u].z; s[3] += v[u].w; }
    }
    for (; k < k1; k++) {
        const int4 v = *(const int4*)(part + (int64_t)k * n + e0);
        s[0] += v.x; s[1] += v.y; s[2] += v.z; s[3] += v.w;
    }
    long long* o = out2 + (int64_t)blockIdx.y * n + e0;
#pragma unroll
    for (int u = 0; u < 4; u++) o[u] = s[u];
}

// few splits: one lane per 4 weights over all splits, sum and max in one pass
// S <= 8 splits, four elements per thread step with every split's 16-byte
// load in flight together; the int64 sums into `out` unless it is null (the
// max partials alone, for a requant that re-sums the splits itself)
template <int S>
__global__ __launch_bounds__(256) void k_wgrad_reduce_flat(const int32_t* __restrict__ part, int64_t n,
                                                           long long* __restrict__ out, uint64_t* pmax)
{
    constexpr int U = S >= 8 ? 1 : 8 / S;      // grid steps per trip: about eight loads in flight
    const int64_t n4 = n >> 2, stride = (int64_t)gridDim.x * 256;
    uint64_t mx = 0;
    for (int64_t j0 = (int64_t)blockIdx.x * 256 + threadIdx.x; j0 < n4; j0 += U * stride) {
        int4 v[U][S];
#pragma unroll
        for (int u = 0; u < U; u++) {
            const int64_t j = j0 + u * stride < n4 ? j0 + u * stride : j0;   // past the end: a repeat
#pragma unroll
            for (int k = 0; k < S; k++) v[u][k] = *(const int4*)(part + (int64_t)k * n + j * 4);
        }
#pragma unroll
        for (int u = 0; u < U; u++) {
            const int64_t j = j0 + u * stride;
            if (j >= n4) break;
            long long s[4] = {0, 0, 0, 0};
#pragma unroll
            for (int k = 0; k < S; k++) { s[0] += v[u][k].x; s[1] += v[u][k].y; s[2] += v[u][k].z; s[3] += v[u][k].w; }
            if (out) {
                *(longlong2*)(out + j * 4) = make_longlong2(s[0], s[1]);
                *(longlong2*)(out + j * 4 + 2) = make_longlong2(s[2], s[3]);
            }
#pragma unroll
            for (int e = 0; e < 4; e++) {
                const uint64_t a = s[e] < 0 ? (uint64_t)(-s[e]) : (uint64_t)s[e];
                mx = a > mx ? a : mx;
            }
        }
    }
    if (pmax) block_store_max_u64(mx, pmax);
}

__global__ __launch_bounds__(256) void k_wgrad_reduce_fin(const long long* __restrict__ out2, int64_t n, int nchunks,
                                                          long long* __restrict__ out, uint64_t* pmax)
{
    const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
    uint64_t mx = 0;
    if (e < n) {
        // eight chunk loads in flight (a loop of dependent single loads waits
        // for each one: up to ~100 round trips for the stem's chunks)
        long long t = 0;
        int c = 0;
        for (; c + 8 <= nchunks; c += 8) {
            long long v[8];
#pragma unroll
            for (int u = 0; u < 8; u++) v[u] = out2[(int64_t)(c + u) * n + e];
#pragma unroll
            for (int u = 0; u < 8; u++) t += v[u];
        }
        for (; c < nchunks; c++) t += out2[(int64_t)c * n + e];
        out[e] = t;
        mx = t < 0 ? (uint64_t)(-t) : (uint64_t)t;
    }
    if (pmax) block_store_max_u64(mx, pmax);
}

// ---------------------------------------------------------------------------
// Backward-weight of the few-channel stem (C = 3, 3x3 / stride 1 or 7x7 /
// stride 2) on v_mfma_i32_32x32x32_i8 with pixels as the reduction: per output
// row of a 16 x 32 tile, A = dy^T (64 output channels x 32 pixels, read with
// ds_read_b64_tr_b8 from the block's dy tile) and B = the 32 pixels' input
// patches ((tap, channel) x pixel, gathered from the LDS halo).  Wave w takes
// rows 4w..4w+3; the four waves' sums are added in LDS and the block writes
// its exact int32 partial [K][R S C] (k_wgrad_reduce adds the blocks in int64).
// ---------------------------------------------------------------------------
template <int C, int R, int S, int ST>
__global__ __launch_bounds__(256) void k_wgrad_stem(const int8_t* __restrict__ dy, const int8_t* __restrict__ x,
                                                   int32_t* __restrict__ part, HaloArgs a)
{
    constexpr int TH = 16, TW = 32, KRED = R * S * C, NKS = (KRED + 31) / 32;
    constexpr int HROWS = (TH - 1) * ST + R, HCOLS = (TW - 1) * ST + S;
    constexpr int NH = HROWS * HCOLS * C;
    constexpr int RD = 80;                                   // LDS bytes per dy pixel row (64 + pad)
    constexpr int DYB = TH * TW * RD;
    __shared__ __attribute__((aligned(16))) int8_t sdy[DYB];
    __shared__ __attribute__((aligned(16))) int8_t shalo[(NH + 15) & ~15];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int l32 = lane & 31, h = lane >> 5;
    const int tx = blockIdx.x % a.tiles_x, t2 = blockIdx.x / a.tiles_x;
    const int ty = t2 % a.tiles_y, n = t2 / a.tiles_y;
    const int oy0 = ty * TH, ox0 = tx * TW, k0 = blockIdx.y * 64;
    const int iy0 = oy0 * ST - a.ph, ix0 = ox0 * ST - a.pw;

    {   // dy tile: 512 pixels x 64 channels, 16-byte pieces, zero outside the output
        int4 v[8];
#pragma unroll
        for (int u = 0; u < 8; u++) {
            const int c = tid + 256 * u, px = c >> 2, part4 = c & 3;
            const int ry = px / TW, rx = px % TW;
            const bool ok = oy0 + ry < a.Ho && ox0 + rx < a.Wo;
            v[u] = ok ? *(const int4*)(dy + (((int64_t)n * a.Ho + oy0 + ry) * a.Wo + ox0 + rx) * a.Nout + k0 +
                                       part4 * 16)
                      : make_int4(0, 0, 0, 0);
        }
        constexpr int PER = (NH + 255) / 256;
        int8_t hv[PER];
#pragma unroll
        for (int u = 0; u < PER; u++) {
            const int i = tid + 256 * u;
            const int hr = i / (HCOLS * C), rem = i - hr * (HCOLS * C);
            const int hc = rem / C, c = rem - hc * C;
            const int iy = iy0 + hr, ix = ix0 + hc;
            const bool ok = i < NH && (unsigned)iy < (unsigned)a.Hs && (unsigned)ix < (unsigned)a.Ws;
            hv[u] = ok ? x[(((int64_t)n * a.Hs + iy) * a.Ws + ix) * C + c] : (int8_t)0;
        }
#pragma unroll
        for (int u = 0; u < 8; u++) {
            const int c = tid + 256 * u;
            *(int4*)&sdy[(c >> 2) * RD + (c & 3) * 16] = v[u];
        }
#pragma unroll
        for (int u = 0; u < PER; u++)
            if (tid + 256 * u < NH) shalo[tid + 256 * u] = hv[u];
    }
    // B gather offsets: this lane's column j = 32 ks + l32 = (tap, channel), -1 past KRED
    int boff[NKS];
#pragma unroll
    for (int ks = 0; ks < NKS; ks++) {
        const int j = 32 * ks + l32;
        const int tap = j / C, c = j - (j / C) * C, r = tap / S, s2 = tap - (tap / S) * S;
        boff[ks] = j < KRED ? (r * HCOLS + s2) * C + c : -1;
    }
    __syncthreads();

    typedef int v16i __attribute__((ext_vector_type(16)));
    v16i acc[2][NKS];
    const int g16 = lane >> 4, sl = lane & 15;
#pragma unroll
    for (int yy = 0; yy < 4; yy++) {
        const int y = 4 * wave + yy;
        // A: channels 32 m + 16 (g16 & 1) + (lane % 16), pixels 16 (g16 >> 1) + 0..15 of row y
        v4i fa[2];
#pragma unroll
        for (int m = 0; m < 2; m++) {
            const int c0 = 32 * m + 16 * (g16 & 1);
            const int px0 = y * TW + 16 * (g16 >> 1);
            const int8_t* p0 = sdy + (px0 + (sl >> 1)) * RD + c0 + 8 * (sl & 1);
            const v2i_t lo = __builtin_amdgcn_ds_read_tr8_b64_v2i32((__attribute__((address_space(3))) v2i_t*)p0);
            const v2i_t hi =
                __builtin_amdgcn_ds_read_tr8_b64_v2i32((__attribute__((address_space(3))) v2i_t*)(p0 + 8 * RD));
            fa[m] = (v4i){lo.x, lo.y, hi.x, hi.y};
        }
#pragma unroll
        for (int ks = 0; ks < NKS; ks++) {
            uint32_t bv[4] = {0, 0, 0, 0};
            if (boff[ks] >= 0) {
                const int8_t* hp = shalo + (y * ST * HCOLS + 16 * h * ST) * C + boff[ks];
#pragma unroll
                for (int b = 0; b < 16; b++) bv[b >> 2] |= (uint32_t)(uint8_t)hp[b * ST * C] << (8 * (b & 3));
            }
            const v4i fb = (v4i){(int)bv[0], (int)bv[1], (int)bv[2], (int)bv[3]};
#pragma unroll
            for (int m = 0; m < 2; m++)
                acc[m][ks] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fa[m], fb, yy ? acc[m][ks] : (v16i){}, 0, 0, 0);
        }
    }
    // sum the four waves in LDS (reusing the dy tile), one 32-column group at a
    // time, and store the block partial
    int32_t* red = (int32_t*)sdy;                           // [4 waves][2][16 values][64 lanes] = 32 KB
    int32_t* outp = part + (int64_t)blockIdx.x * a.Nout * KRED;
#pragma unroll
    for (int ks = 0; ks < NKS; ks++) {
        __syncthreads();
#pragma unroll
        for (int m = 0; m < 2; m++)
#pragma unroll
            for (int v = 0; v < 16; v++) red[((wave * 2 + m) * 16 + v) * 64 + lane] = acc[m][ks][v];
        __syncthreads();
        for (int e = tid; e < 2 * 16 * 64; e += 256) {
            const int m = e >> 10, v = (e >> 6) & 15, ln = e & 63;
            int32_t t = 0;
#pragma unroll
            for (int w = 0; w < 4; w++) t += red[((w * 2 + m) * 16 + v) * 64 + ln];
            const int ch = 32 * m + 8 * (v >> 2) + 4 * (ln >> 5) + (v & 3);
            const int col = 32 * ks + (ln & 31);
            if (col < KRED) outp[(int64_t)(k0 + ch) * KRED + col] = t;
        }
    }
}

#ifndef ISEG_WGRAD_BLOCKS
#define ISEG_WGRAD_BLOCKS 384      // target blocks of a split backward-weight launch
#endif

int64_t wgrad_splits(int64_t NPQ, int64_t tiles, int64_t* pps_out)
{
    int64_t splits = ceil_div64(ISEG_WGRAD_BLOCKS, tiles);
    int64_t min_splits = ceil_div64(NPQ, kWgradSplit);
    int64_t max_splits = ceil_div64(NPQ, 64 * 4);
    if (splits > max_splits) splits = max_splits;
    if (splits < min_splits) splits = min_splits;
    if (splits > 65535) splits = 65535;
    int64_t pps = ceil_div64(ceil_div64(NPQ, splits), 64) * 64;
    if (pps > kWgradSplit) pps = kWgradSplit;
    *pps_out = pps;
    return ceil_div64(NPQ, pps);
}

#ifndef ISEG_WGRAD_TAPS_BLOCKS
#define ISEG_WGRAD_TAPS_BLOCKS 128 // target blocks of the all-taps backward-weight launch (it runs beside the main chain: half the chip)
#endif
// shapes the all-taps kernel covers (the operand alignment is checked at launch):
// filters of 9 taps (3x3); one wave per tap keeps a 576-thread block at three
// waves per SIMD with no spills
bool wgrad_taps_shape(int64_t NPQ, int64_t K, int64_t C, int64_t RS)
{
    return NPQ > 0 && C % 64 == 0 && K % 64 == 0 && RS == 9;
}

// split count and pixels per split of the all-taps kernel; the int32 partial
// of one split stays exact because a split sums at most kWgradSplit products
int64_t wgrad_taps_splits(int64_t NPQ, int64_t K, int64_t C, int64_t* pps_out)
{
    int64_t tiles = (C / 64) * (K / 64);
    int64_t splits = ceil_div64(ISEG_WGRAD_TAPS_BLOCKS, tiles);
    int64_t min_splits = ceil_div64(NPQ, kWgradSplit);
    int64_t max_splits = ceil_div64(NPQ, 64 * 4);
    if (splits > max_splits) splits = max_splits;
    if (splits < min_splits) splits = min_splits;
    if (splits > 65535) splits = 65535;
    int64_t pps = ceil_div64(ceil_div64(NPQ, splits), 64) * 64;
    if (pps > kWgradSplit) pps = kWgradSplit;
    *pps_out = pps;
    return ceil_div64(NPQ, pps);
}

// chunks of the splits reduced by separate blocks: enough blocks for the chip
// when the weight tensor alone gives too few, each chunk still >= 8 splits
int wgrad_reduce_chunks(int64_t n, int64_t splits)
{
    const int64_t bx = ceil_div64(n, 1024);
    if (bx >= 512 || splits < 16) return 1;
    int64_t c = ceil_div64(1024, bx);
    const int64_t cmax = splits / 8;
    c = c < cmax ? c : cmax;
    return (int)(c < 1 ? 1 : c);
}

size_t wgrad_taps_part_bytes(int64_t NPQ, int64_t K, int64_t C, int64_t RS)
{
    if (!wgrad_taps_shape(NPQ, K, C, RS)) return 0;
    int64_t pps;
    int64_t splits = wgrad_taps_splits(NPQ, K, C, &pps);
    const int64_t n = K * RS * C;
    const int nch = wgrad_reduce_chunks(n, splits);
    return align256((size_t)(splits * n) * 4) + (nch > 1 ? align256((size_t)(nch * n) * 8) : 0);
}

// all-taps launch: partials into `part`, then their int64 sum into a.acc (every
// element written, no fill needed) and its max |.| into maxp when given
// int64 sums of `splits` int32 partials [splits][n] (n % 4 == 0) into out and,
// when pmax is set, per-block max |sum| partials (their count into *npmax);
// the two-level variant keeps its chunk sums right after the partials
bool wgrad_flat_ok(int64_t n, int64_t splits) { return splits >= 1 && splits <= 8 && n % 4 == 0; }

int launch_wgrad_reduce(const int32_t* part, int64_t n, int64_t splits, long long* out, uint64_t* pmax,
                        int64_t* npmax, hipStream_t s)
{
    const int nch = wgrad_reduce_chunks(n, splits);
    if (nch > 1) {
        long long* out2 = (long long*)((char*)part + align256((size_t)(splits * n) * 4));
        const int chunk = (int)ceil_div64(splits, nch);
        hipLaunchKernelGGL(k_wgrad_reduce_part, dim3((unsigned)ceil_div64(n, 1024), (unsigned)nch), dim3(256), 0, s,
                           part, n, (int)splits, chunk, out2);
        int rc = launch_ok();
        if (rc) return rc;
        if (npmax) *npmax = ceil_div64(n, 256);
        hipLaunchKernelGGL(k_wgrad_reduce_fin, dim3((unsigned)ceil_div64(n, 256)), dim3(256), 0, s,
                           (const long long*)out2, n, nch, out, pmax);
        return launch_ok();
    }
    if (wgrad_flat_ok(n, splits) && (((uintptr_t)out) & 15) == 0) {
        // a capped grid: the requant that follows reduces every max partial in each block
        const unsigned nb = (unsigned)std::min<int64_t>(ceil_div64(n / 4, 256), 512);
        if (npmax) *npmax = nb;
        switch (splits) {
#define ISEG_RF(S) case S: hipLaunchKernelGGL(k_wgrad_reduce_flat<S>, dim3(nb), dim3(256), 0, s, part, n, out, pmax); break;
        ISEG_RF(1) ISEG_RF(2) ISEG_RF(3) ISEG_RF(4) ISEG_RF(5) ISEG_RF(6) ISEG_RF(7) ISEG_RF(8)
#undef ISEG_RF
        }
        return launch_ok();
    }
    if (!out) return ISEG_ERR_ARG;
    if (npmax) *npmax = ceil_div64(n, 256);
    hipLaunchKernelGGL(k_wgrad_reduce, dim3((unsigned)ceil_div64(n, 256)), dim3(64 * kRedWaves), 0, s, part, n,
                       (int)splits, out, pmax);
    return launch_ok();
}

// The split reduction ahead of Q_G.  When `qg` is given and the splits allow
// the flat reduce, only the max partials are formed and *qg = splits: the
// requant re-sums the int32 splits itself (launch_requant_splits), so the
// int64 sums are never written; otherwise the int64 sums go to `out`, *qg = 0.
int launch_wgrad_reduce_qg(const int32_t* part, int64_t n, int64_t splits, long long* out, uint64_t* pmax,
                           int64_t* npmax, hipStream_t s, int* qg)
{
    const bool fuse = qg && pmax && wgrad_flat_ok(n, splits);
    if (qg) *qg = fuse ? (int)splits : 0;
    return launch_wgrad_reduce(part, n, splits, fuse ? nullptr : out, pmax, npmax, s);
}

// max-partial count of launch_wgrad_reduce for a shape (workspace sizing)
int64_t wgrad_reduce_npmax(int64_t n) { return ceil_div64(n, 256); }

// all-taps launch: partials into `part`, then their int64 sum into a.acc (every
// element written, no fill needed) and its max |.| partials into pmax when given
int launch_wgrad_taps(WgradArgs a, int32_t* part, uint64_t* pmax, int64_t* npmax, hipStream_t s, int* qg)
{
    const int RS = a.R * a.S;
    int64_t splits = wgrad_taps_splits(a.NPQ, a.K, a.C, &a.pix_per_split);
    if (RS != 9) return ISEG_ERR_UNSUPPORTED;
    const size_t lds = wgrad_taps_lds(9);
    if (!lds_limit((const void*)k_conv_wgrad_taps<9>, lds))
        return ISEG_ERR_DEVICE;
    dim3 grid((unsigned)((a.C / 64) * (a.K / 64)), (unsigned)splits);
    ISEG_TIMED_LAUNCH(ISEG_KID_CONV_WGRAD, s, k_conv_wgrad_taps<9>, grid, dim3(64 * 9), lds, s, a, part);
    int rc = launch_ok();
    if (rc) return rc;
    return launch_wgrad_reduce_qg(part, (int64_t)a.K * a.RSC, splits, (long long*)a.acc, pmax, npmax, s, qg);
}

// the transposed-operand kernel over split pixel ranges: int32 partials per
// split stored into `part`, summed like the all-taps kernel's (C % 64 == 0,
// K % 64 == 0, 16-byte aligned operands)
bool wgrad_tr_ok(const WgradArgs& a)
{
    const int64_t nimg = a.P > 0 && a.Q > 0 ? a.NPQ / ((int64_t)a.P * a.Q) : 0;
    return a.NPQ > 0 && a.C % 64 == 0 && a.K % 64 == 0 && (((uintptr_t)a.x | (uintptr_t)a.dy) & 15) == 0 &&
           nimg * a.H * a.W * a.C < ((int64_t)1 << 31) && a.NPQ * a.K < ((int64_t)1 << 31);
}

int64_t wgrad_tr_splits(const WgradArgs& a, int64_t* pps)
{
    const int BMt = a.K % 128 == 0 ? 128 : 64;
    const int RS = a.R * a.S;
    const int TAPS = RS > 1 ? 2 : 1;
    const int ntg = (RS + TAPS - 1) / TAPS;
    const int64_t tiles = (int64_t)ntg * (a.C / 64) * (a.K / BMt);
    return wgrad_splits(a.NPQ, tiles, pps);
}

size_t wgrad_tr_part_bytes(int64_t NPQ, int64_t K, int64_t C, int64_t RS)
{
    if (NPQ <= 0 || C % 64 || K % 64) return 0;
    WgradArgs a{};
    a.NPQ = NPQ; a.K = (int32_t)K; a.C = (int32_t)C; a.R = (int32_t)RS; a.S = 1;
    int64_t pps;
    const int64_t splits = wgrad_tr_splits(a, &pps);
    const int64_t n = K * RS * C;
    const int nch = wgrad_reduce_chunks(n, splits);
    return align256((size_t)(splits * n) * 4) + (nch > 1 ? align256((size_t)(nch * n) * 8) : 0);
}

int launch_wgrad_tr_split(WgradArgs a, int32_t* part, uint64_t* pmax, int64_t* npmax, hipStream_t s, int* qg)
{
    const int BMt = a.K % 128 == 0 ? 128 : 64;
    const int RS = a.R * a.S;
    const int TAPS = RS > 1 ? 2 : 1;
    const int ntg = (RS + TAPS - 1) / TAPS;
    const int64_t splits = wgrad_tr_splits(a, &a.pix_per_split);
    a.part = part;
    dim3 grid((unsigned)(ntg * (a.C / 64)), (unsigned)(a.K / BMt), (unsigned)splits);
    if (BMt == 128 && TAPS == 2)
        hipLaunchKernelGGL((k_conv_wgrad_tr<128, 2>), grid, dim3(256), 0, s, a);
    else if (BMt == 128)
        hipLaunchKernelGGL((k_conv_wgrad_tr<128, 1>), grid, dim3(256), 0, s, a);
    else if (TAPS == 2)
        hipLaunchKernelGGL((k_conv_wgrad_tr<64, 2>), grid, dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL((k_conv_wgrad_tr<64, 1>), grid, dim3(256), 0, s, a);
    int rc = launch_ok();
    if (rc) return rc;
    return launch_wgrad_reduce_qg(part, (int64_t)a.K * a.RSC, splits, (long long*)a.acc, pmax, npmax, s, qg);
}

int launch_wgrad(WgradArgs a, hipStream_t s)
{
    if (wgrad_tr_ok(a)) {
        const int BMt = a.K % 128 == 0 ? 128 : 64;
        const int RS = a.R * a.S;
        const int TAPS = RS > 1 ? 2 : 1;
        const int ntg = (RS + TAPS - 1) / TAPS;
        int64_t tiles = (int64_t)ntg * (a.C / 64) * (a.K / BMt);
        int64_t splits = wgrad_splits(a.NPQ, tiles, &a.pix_per_split);
        dim3 grid((unsigned)(ntg * (a.C / 64)), (unsigned)(a.K / BMt), (unsigned)splits);
        if (BMt == 128 && TAPS == 2)
            ISEG_TIMED_LAUNCH(ISEG_KID_CONV_WGRAD, s, (k_conv_wgrad_tr<128, 2>), grid, dim3(256), 0, s, a);
        else if (BMt == 128)
            ISEG_TIMED_LAUNCH(ISEG_KID_CONV_WGRAD, s, (k_conv_wgrad_tr<128, 1>), grid, dim3(256), 0, s, a);
        else if (TAPS == 2)
            ISEG_TIMED_LAUNCH(ISEG_KID_CONV_WGRAD, s, (k_conv_wgrad_tr<64, 2>), grid, dim3(256), 0, s, a);
        else
            ISEG_TIMED_LAUNCH(ISEG_KID_CONV_WGRAD, s, (k_conv_wgrad_tr<64, 1>), grid, dim3(256), 0, s, a);
        return launch_ok();
    }
    if (a.NPQ > 0 && a.C % 64 == 0 && a.K % 4 == 0 &&
        (((uintptr_t)a.x | (uintptr_t)a.dy) & 3) == 0) {
        const int BMt = a.K >= 128 ? 128 : 64;
        int64_t tiles = (int64_t)a.R * a.S * (a.C / 64) * ceil_div64(a.K, BMt);
        int64_t splits = wgrad_splits(a.NPQ, tiles, &a.pix_per_split);
        dim3 grid((unsigned)(a.R * a.S * (a.C / 64)), (unsigned)ceil_div64(a.K, BMt), (unsigned)splits);
        if (BMt == 128)
            ISEG_TIMED_LAUNCH(ISEG_KID_CONV_WGRAD, s, k_conv_wgrad_tap<128>, grid, dim3(256), 0, s, a);
        else
            ISEG_TIMED_LAUNCH(ISEG_KID_CONV_WGRAD, s, k_conv_wgrad_tap<64>, grid, dim3(256), 0, s, a);
        return launch_ok();
    }
    return launch_wgrad_generic(a, s);
}

int launch_wgrad_generic(WgradArgs a, hipStream_t s)
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
// room for per-block max partials of any path the output of rows x cols can take
size_t conv_pmax_bytes(int64_t rows, int64_t cols, const HaloPlan& hp, int64_t N, int64_t Ho, int64_t Wo)
{
    int64_t nb = ceil_div64(rows, 128) * ceil_div64(cols, 64);
    if (hp.ok) {
        const int64_t nh = N * hp.tiles_y * hp.tiles_x * (cols / 64);
        nb = nb > nh ? nb : nh;
    }
    const int64_t nm = N * ceil_div64(Ho, kM32TH) * ceil_div64(Wo, kM32TW) * ceil_div64(cols, 64);
    nb = nb > nm ? nb : nm;
    return align256((size_t)nb * 8);
}

static size_t conv_fwd_core_ws(const iseg_conv_geom* g, int32_t out_mode)
{
    int64_t P, Q;
    if (!geom_ok(g, &P, &Q)) return 0;
    size_t s = 256;
    if (out_mode == ISEG_OUT_Q8) {
        size_t big = align256((size_t)(g->N * P * Q * g->K) * 4);
        const size_t s16 = staged_ws_bytes(g->N * P * Q, g->K);
        big = big > s16 ? big : s16;
        const DmaPlan dp = dma_plan(g->N * P * Q, (int32_t)g->K, (int32_t)(padded_c(g->C) * g->R * g->S), true);
        const size_t sk = dma_split_bytes(dp, g->N * P * Q, (int32_t)g->K);
        big = big > sk ? big : sk;
        const HaloPlan hp = halo_plan(g->N, P, Q, g->C, g->K, (int)g->R, (int)g->S, g->stride_h, g->stride_w,
                                      g->dil_h, g->dil_w);
        if (hp.ok) {
            const size_t sh = halo_staged_ws_bytes(hp, g->N, P, Q, g->K);
            big = big > sh ? big : sh;
        }
        s += big + conv_pmax_bytes(g->N * P * Q, g->K, hp, g->N, P, Q);
    }
    int64_t Cp = padded_c(g->C);
    if (Cp != g->C)
        s += align256((size_t)(g->N * g->H * g->W * Cp)) + align256((size_t)(g->K * g->R * g->S * Cp));
    return s;
}

static int conv_fwd_core(const int8_t* x, const int32_t* x_exp, const int8_t* w, const int32_t* w_exp,
                         const iseg_conv_geom* g, int32_t out_mode, void* y, int32_t* y_exp,
                         void* ws, size_t ws_bytes, int32_t* dev_status, hipStream_t stream)
{
    (void)dev_status;
    int64_t P, Q;
    if (!geom_ok(g, &P, &Q)) return ISEG_ERR_SHAPE;
    if (out_mode != ISEG_OUT_Q8 && out_mode != ISEG_OUT_RAW) return ISEG_ERR_ARG;
    if (!x_exp || !w_exp || !y_exp || (g->N > 0 && (!x || !w || !y))) return ISEG_ERR_ARG;
    if (g->C * g->R * g->S > kMaxKred) return ISEG_ERR_UNSUPPORTED;
    if (!ws || ws_bytes < conv_fwd_core_ws(g, out_mode)) return ISEG_ERR_WORKSPACE;
    // ws: [max][per-block max partials][output staging][padded operands]
    unsigned long long* maxp = (unsigned long long*)ws;
    const int64_t Cp = padded_c(g->C);
    const HaloPlan hp = halo_plan(g->N, P, Q, Cp, g->K, (int)g->R, (int)g->S, g->stride_h, g->stride_w,
                                  g->dil_h, g->dil_w);
    char* wp = (char*)ws + 256;
    uint64_t* pmax = nullptr;
    int32_t* acc = (int32_t*)y;
    if (out_mode == ISEG_OUT_Q8) {
        pmax = (uint64_t*)wp;
        wp += conv_pmax_bytes(g->N * P * Q, g->K, hp, g->N, P, Q);
        acc = (int32_t*)wp;
        size_t big = align256((size_t)(g->N * P * Q * g->K) * 4);
        const size_t s16 = staged_ws_bytes(g->N * P * Q, g->K);
        big = big > s16 ? big : s16;
        const DmaPlan dp = dma_plan(g->N * P * Q, (int32_t)g->K, (int32_t)(Cp * g->R * g->S), true);
        const size_t sk = dma_split_bytes(dp, g->N * P * Q, (int32_t)g->K);
        big = big > sk ? big : sk;
        if (hp.ok) {
            const size_t sh = halo_staged_ws_bytes(hp, g->N, P, Q, g->K);
            big = big > sh ? big : sh;
        }
        wp += big;
    }
    int rc;
    const int stem = stem_kind(g->C, (int)g->R, (int)g->S, g->stride_h, g->stride_w, g->dil_h, g->dil_w, g->K);
    if (stem && g->N > 0) {
        conv_plan_set("stem");
        HaloArgs h{};
        h.src = x; h.wmat = w; h.out = (int32_t*)y;
        h.N = (int32_t)g->N; h.Hs = (int32_t)g->H; h.Ws = (int32_t)g->W; h.Ci = (int32_t)g->C;
        h.Ho = (int32_t)P; h.Wo = (int32_t)Q; h.Nout = (int32_t)g->K;
        h.ph = g->pad_h; h.pw = g->pad_w; h.dh = 1; h.dw = 1;
        if (out_mode == ISEG_OUT_RAW) {
            if ((rc = launch_stem(stem, h, EPI_RAW, ISEG_KID_CONV_FWD, stream))) return rc;
            hipLaunchKernelGGL(k_exp_sum, dim3(1), dim3(1), 0, stream, y_exp, x_exp, w_exp);
            return launch_ok();
        }
        h.pmax = pmax;
        h.npmax = (int64_t)g->N * ceil_div64(P, 16) * ceil_div64(Q, 32) * (g->K / 64);
        if ((rc = launch_stem(stem, h, EPI_MAX, ISEG_KID_CONV_FWD, stream))) return rc;
        h.out8 = (int8_t*)y; h.exp_a = x_exp; h.exp_b = w_exp; h.out_exp = y_exp;
        return launch_stem(stem, h, EPI_Q8, ISEG_KID_CONV_FWD, stream);
    }
    // small C: zero-pad channels to a multiple of 16 for the vector path
    const int8_t* xs = x;
    const int8_t* wsrc = w;
    if (Cp != g->C) {
        int8_t* xp = (int8_t*)wp;
        wp += align256((size_t)(g->N * g->H * g->W * Cp));
        int8_t* wpd = (int8_t*)wp;
        if ((rc = launch_pad(x, xp, g->N * g->H * g->W, g->C, Cp, stream))) return rc;
        if ((rc = launch_pad(w, wpd, g->K * g->R * g->S, g->C, Cp, stream))) return rc;
        xs = xp;
        wsrc = wpd;
    }
    IgemmArgs a{};
    a.src = xs; a.wmat = wsrc; a.out = acc; a.pmax = pmax;
    a.out16 = nullptr; a.tshift = nullptr;
    a.Mrows = g->N * P * Q;
    a.Nout = (int32_t)g->K; a.Kred = (int32_t)(Cp * g->R * g->S); a.Ci = (int32_t)Cp;
    a.Hs = (int32_t)g->H; a.Ws = (int32_t)g->W; a.Ho = (int32_t)P; a.Wo = (int32_t)Q;
    a.R = (int32_t)g->R; a.S = (int32_t)g->S;
    a.sh = g->stride_h; a.sw = g->stride_w; a.ph = g->pad_h; a.pw = g->pad_w;
    a.dh = g->dil_h; a.dw = g->dil_w;
    const M32Plan mp = m32_plan(g->N, P, Q, Cp, g->K, (int)g->R, (int)g->S, g->stride_h, g->stride_w, g->dil_h,
                                g->dil_w);
    if (mp.ok && (((uintptr_t)xs | (uintptr_t)wsrc | (uintptr_t)y) & 15) == 0) {
        conv_plan_set("m32");
        HaloArgs h{};
        h.src = xs; h.wmat = wsrc; h.out = (int32_t*)y;
        h.N = (int32_t)g->N; h.Hs = (int32_t)g->H; h.Ws = (int32_t)g->W; h.Ci = (int32_t)Cp;
        h.Ho = (int32_t)P; h.Wo = (int32_t)Q; h.Nout = (int32_t)g->K;
        h.ph = g->pad_h; h.pw = g->pad_w; h.dh = g->dil_h; h.dw = g->dil_w;
        if (out_mode == ISEG_OUT_RAW) {
            if ((rc = launch_m32(mp, h, EPI_RAW, ISEG_KID_CONV_FWD, stream))) return rc;
            hipLaunchKernelGGL(k_exp_sum, dim3(1), dim3(1), 0, stream, y_exp, x_exp, w_exp);
            return launch_ok();
        }
        return m32_q8(mp, h, ISEG_KID_CONV_FWD, x_exp, w_exp, (int8_t*)y, y_exp, pmax, stream);
    }
    const PersistPlan pp = persist_plan(g->N, P, Q, Cp, g->K, (int)g->R, (int)g->S, g->stride_h, g->stride_w,
                                        g->dil_h, g->dil_w);
    if (pp.ok && (((uintptr_t)xs | (uintptr_t)wsrc | (uintptr_t)y) & 15) == 0) {
        conv_plan_set("persist");
        HaloArgs h{};
        h.src = xs; h.wmat = wsrc; h.out = (int32_t*)y;
        h.N = (int32_t)g->N; h.Hs = (int32_t)g->H; h.Ws = (int32_t)g->W; h.Ci = (int32_t)Cp;
        h.Ho = (int32_t)P; h.Wo = (int32_t)Q; h.Nout = (int32_t)g->K;
        h.ph = g->pad_h; h.pw = g->pad_w; h.dh = g->dil_h; h.dw = g->dil_w;
        if (out_mode == ISEG_OUT_RAW) {
            if ((rc = launch_persist(pp, h, EPI_RAW, ISEG_KID_CONV_FWD, stream))) return rc;
            hipLaunchKernelGGL(k_exp_sum, dim3(1), dim3(1), 0, stream, y_exp, x_exp, w_exp);
            return launch_ok();
        }
        return persist_q8(pp, h, ISEG_KID_CONV_FWD, x_exp, w_exp, (int8_t*)y, y_exp, pmax, stream);
    }
    if (hp.ok && (((uintptr_t)xs | (uintptr_t)wsrc | (uintptr_t)y | (uintptr_t)acc) & 15) == 0) {
        conv_plan_set("halo");
        HaloArgs h{};
        h.src = xs; h.wmat = wsrc; h.out = acc;
        h.out16 = out_mode == ISEG_OUT_Q8 ? (int16_t*)acc : nullptr;
        h.tshift = (uint8_t*)acc + align256((size_t)(a.Mrows * a.Nout) * 2);
        h.N = (int32_t)g->N; h.Hs = (int32_t)g->H; h.Ws = (int32_t)g->W; h.Ci = (int32_t)Cp;
        h.Ho = (int32_t)P; h.Wo = (int32_t)Q; h.Nout = (int32_t)g->K;
        h.ph = g->pad_h; h.pw = g->pad_w; h.dh = g->dil_h; h.dw = g->dil_w;
        if (out_mode == ISEG_OUT_RAW) {
            if ((rc = launch_halo(hp, h, EPI_RAW, ISEG_KID_CONV_FWD, stream))) return rc;
            hipLaunchKernelGGL(k_exp_sum, dim3(1), dim3(1), 0, stream, y_exp, x_exp, w_exp);
            return launch_ok();
        }
        return halo_q8(hp, h, ISEG_KID_CONV_FWD, x_exp, w_exp, (int8_t*)y, y_exp, maxp, pmax, a.Mrows, stream);
    }
    if (igemm_dma_ok(a) && ((uintptr_t)y & 15) == 0)
        return igemm_dma_run<MODE_FWD>(a, out_mode, x_exp, w_exp, y, y_exp, pmax, acc, stream);
    int64_t nblk = 0;
    conv_plan_set("igemm");
    if ((rc = launch_igemm<MODE_FWD>(a, stream, &nblk))) return rc;
    if (out_mode == ISEG_OUT_RAW) {
        hipLaunchKernelGGL(k_exp_sum, dim3(1), dim3(1), 0, stream, y_exp, x_exp, w_exp);
        return launch_ok();
    }
    return launch_requant_apply(acc, ISEG_I32, a.Mrows * a.Nout, x_exp, w_exp, 0, 8, 0, 1,
                                0, 0, 0, ISEG_I8, y, y_exp, nullptr, stream, pmax, nblk);
}

// ---------------------------------------------------------------------------
// Backward-data of a strided conv with few output-gradient channels (K < 64,
// or K = 64 at stride products >= 4), e.g. the bilinear upsampling layers of
// FCN (transposed convs of stride 2 and 8 over the class scores), by phase
// decomposition.  Input pixel h receives only the taps r = ((h + pad) mod
// stride) + t * stride, from dy row p = floor((h + pad) / stride) - t, so all
// pixels of one phase ((h + pad) mod stride_h, (w + pad) mod stride_w) share
// their taps.  A block takes a 16 x 16 tile of one phase's pixels, stages the
// dy rows they read in LDS (K padded to Kp, a multiple of 8, with zeros) and
// sums with v_dot4 over 4 dy channels at a time against the weights
// repacked as [R][S][Cp][Kp] (one address for the whole block: scalar
// loads); eight output channels per thread, blockIdx.y picks the group.
// Only the taps that meet real dy entries are computed, where the implicit
// GEMM multiplies stride_h * stride_w times as many products, most of them
// with the zeros between the dy rows.
// ---------------------------------------------------------------------------
constexpr int kTcTile = 16, kTcCB = 8, kTcMaxTaps = 4, kTcMaxKp = 64;

struct TconvArgs {
    const int8_t* dy;          // [N][P][Q][K]
    const int8_t* wp;          // [R][S][Cp][Kp]
    int32_t* out;              // EPI_RAW: [N][H][W][C] int32
    int8_t* out8;              // EPI_Q8: [N][H][W][C] codes
    uint64_t* pmax;            // one max partial per block
    int64_t npmax;
    const int32_t* exp_a;
    const int32_t* exp_b;
    int32_t* out_exp;
    int32_t N, H, W, C, K, Kp, Cp, P, Q, R, S, sh, sw, ph, pw;
    int32_t tiles_h, tiles_w;  // 16 x 16 tiles over ceil(H / sh) x ceil(W / sw) phase pixels
};

struct TconvPlan {
    bool ok = false;
    int32_t Kp = 0, Cp = 0, tiles_h = 0, tiles_w = 0;
    int64_t gx = 0, gy = 0;
};

static TconvPlan tconv_plan(const iseg_conv_geom* g)
{
    TconvPlan t;
    if (g->dil_h != 1 || g->dil_w != 1 || (g->stride_h == 1 && g->stride_w == 1)) return t;
    if (g->K > 64 || (g->K == 64 && g->stride_h * g->stride_w < 4)) return t;
    if (ceil_div64(g->R, g->stride_h) > kTcMaxTaps || ceil_div64(g->S, g->stride_w) > kTcMaxTaps) return t;
    t.Kp = (int32_t)((g->K + 7) & ~(int64_t)7);
    t.Cp = (int32_t)((g->C + kTcCB - 1) / kTcCB * kTcCB);
    t.tiles_h = (int32_t)ceil_div64(ceil_div64(g->H, g->stride_h), kTcTile);
    t.tiles_w = (int32_t)ceil_div64(ceil_div64(g->W, g->stride_w), kTcTile);
    t.gx = g->N * g->stride_h * g->stride_w * t.tiles_h * t.tiles_w;
    t.gy = t.Cp / kTcCB;
    t.ok = t.gx >= 1 && t.gx < ((int64_t)1 << 31) && t.gy < 65536 && g->N * g->H * g->W * g->C < ((int64_t)1 << 40);
    return t;
}

static size_t tconv_ws_bytes(const iseg_conv_geom* g, const TconvPlan& t)
{
    return align256((size_t)(g->R * g->S * t.Cp * t.Kp)) + align256((size_t)(t.gx * t.gy) * 8);
}

// wp[(r S + s) Cp + c][k] = w[k][r][s][c], zero for k >= K or c >= C
__global__ __launch_bounds__(256) void k_tconv_pack(const int8_t* __restrict__ w, int8_t* __restrict__ wp,
                                                    int32_t K, int32_t RS, int32_t C, int32_t Kp, int32_t Cp)
{
    const int64_t n = (int64_t)RS * Cp * Kp;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        const int32_t k = (int32_t)(i % Kp);
        const int64_t rc = i / Kp;
        const int32_t c = (int32_t)(rc % Cp), rs = (int32_t)(rc / Cp);
        wp[i] = (k < K && c < C) ? w[((int64_t)k * RS + rs) * C + c] : (int8_t)0;
    }
}

template <int EPI>
__global__ __launch_bounds__(256) void k_tconv_phase(TconvArgs a)
{
    constexpr int HMAX = kTcTile + kTcMaxTaps - 1;
    __shared__ __attribute__((aligned(16))) int32_t sdy[HMAX * HMAX * (kTcMaxKp / 4)];
    const int tid = threadIdx.x, ty = tid >> 4, tx = tid & 15;
    int64_t b = blockIdx.x;
    const int tw_i = (int)(b % a.tiles_w);
    b /= a.tiles_w;
    const int th_i = (int)(b % a.tiles_h);
    b /= a.tiles_h;
    const int phw = (int)(b % a.sw);
    b /= a.sw;
    const int phh = (int)(b % a.sh);
    const int n = (int)(b / a.sh);
    uint64_t gmax = 0;
    if (EPI == EPI_Q8) gmax = reduce_partials_u64(a.pmax, a.npmax);
    // taps of this phase and the first phase row / column of the tile
    const int Th = phh < a.R ? (a.R - phh + a.sh - 1) / a.sh : 0;
    const int Tw = phw < a.S ? (a.S - phw + a.sw - 1) / a.sw : 0;
    const int mh0 = (max(0, a.ph - phh) + a.sh - 1) / a.sh + th_i * kTcTile;
    const int mw0 = (max(0, a.pw - phw) + a.sw - 1) / a.sw + tw_i * kTcTile;
    const int KW = a.Kp >> 2;
    const int HR = kTcTile + (Th > 0 ? Th - 1 : 0), HC = kTcTile + (Tw > 0 ? Tw - 1 : 0);
    const int p0 = mh0 - (Th > 0 ? Th - 1 : 0), q0 = mw0 - (Tw > 0 ? Tw - 1 : 0);
    int32_t acc[kTcCB];
#pragma unroll
    for (int j = 0; j < kTcCB; j++) acc[j] = 0;
    if (Th > 0 && Tw > 0) {
        // the dy rows p0 .. p0 + HR - 1, columns q0 .. q0 + HC - 1 (zero outside)
        const bool words = (a.K & 3) == 0 && ((uintptr_t)a.dy & 3) == 0;
        const int total = HR * HC * KW;
        for (int i = tid; i < total; i += 256) {
            const int kw = i % KW, pix = i / KW;
            const int p = p0 + pix / HC, q = q0 + pix % HC;
            int32_t v = 0;
            if (p >= 0 && p < a.P && q >= 0 && q < a.Q) {
                const int8_t* src = a.dy + (((int64_t)n * a.P + p) * a.Q + q) * a.K;
                const int k = kw * 4;
                if (words) {
                    if (k < a.K) v = *(const int32_t*)(src + k);
                } else {
                    uint32_t u = 0;
#pragma unroll
                    for (int e = 0; e < 4; e++)
                        if (k + e < a.K) u |= (uint32_t)(uint8_t)src[k + e] << (8 * e);
                    v = (int32_t)u;
                }
            }
            sdy[i] = v;
        }
        __syncthreads();
        const int c0 = blockIdx.y * kTcCB;
        for (int th = 0; th < Th; th++)
            for (int tw = 0; tw < Tw; tw++) {
                const int r = phh + th * a.sh, sx = phw + tw * a.sw;
                const int32_t* wrow = (const int32_t*)(a.wp + (((int64_t)r * a.S + sx) * a.Cp + c0) * a.Kp);
                const int32_t* srow = sdy + ((ty + Th - 1 - th) * HC + (tx + Tw - 1 - tw)) * KW;
                for (int kw = 0; kw < KW; kw += 2) {
                    const int2 v = *(const int2*)(srow + kw);
#pragma unroll
                    for (int j = 0; j < kTcCB; j++) {
                        acc[j] = __builtin_amdgcn_sdot4(v.x, wrow[j * KW + kw], acc[j], false);
                        acc[j] = __builtin_amdgcn_sdot4(v.y, wrow[j * KW + kw + 1], acc[j], false);
                    }
                }
            }
    }
    const int h = (mh0 + ty) * a.sh + phh - a.ph, w = (mw0 + tx) * a.sw + phw - a.pw;
    const bool valid = h < a.H && w < a.W;            // h, w >= 0 by the choice of mh0, mw0
    const int c0 = blockIdx.y * kTcCB;
    const int64_t o = (((int64_t)n * a.H + h) * a.W + w) * a.C + c0;
    const int nc = a.C - c0 < kTcCB ? a.C - c0 : kTcCB;
    if (EPI == EPI_RAW) {
        if (valid)
#pragma unroll
            for (int j = 0; j < kTcCB; j++)
                if (j < nc) a.out[o + j] = acc[j];
        return;
    }
    if (EPI == EPI_MAX) {
        uint32_t mx = 0;
#pragma unroll
        for (int j = 0; j < kTcCB; j++) {
            const uint32_t av = (valid && j < nc) ? (uint32_t)(acc[j] < 0 ? -acc[j] : acc[j]) : 0u;
            mx = av > mx ? av : mx;
        }
        block_store_max_u64(mx, a.pmax);
        return;
    }
    // EPI_Q8: SQ codes with r = bitlen(global max) - 7 (half-up rounding)
    const int rq = gmax ? (64 - __builtin_clzll(gmax)) - 7 : 0;
    if (blockIdx.x == 0 && blockIdx.y == 0 && tid == 0) *a.out_exp = *a.exp_a + *a.exp_b + rq;
    const int rs = rq > 0 ? rq - 1 : 0, ls = rq > 0 ? 0 : -rq;
    if (valid)
#pragma unroll
        for (int j = 0; j < kTcCB; j++) {
            if (j >= nc) break;
            int32_t c = rq > 0 ? ((acc[j] >> rs) + 1) >> 1 : acc[j] << ls;
            c = c > 127 ? 127 : (c < -127 ? -127 : c);
            a.out8[o + j] = (int8_t)c;
        }
}

template <int EPI>
static int launch_tconv_e(const TconvPlan& t, const TconvArgs& a, hipStream_t s)
{
    ISEG_TIMED_LAUNCH(ISEG_KID_CONV_BWD_DATA, s, k_tconv_phase<EPI>, dim3((unsigned)t.gx, (unsigned)t.gy), dim3(256),
                      0, s, a);
    return launch_ok();
}

// the phase path of backward-data: raw sums, or a max pass and a code pass
// (the sums are recomputed: K * taps products per output are cheaper to redo
// than an int32 round trip through HBM)
static int tconv_run(const TconvPlan& t, const iseg_conv_geom* g, int64_t P, int64_t Q, const int8_t* dy,
                     const int32_t* dy_exp, const int8_t* w, const int32_t* w_exp, int32_t out_mode, void* dx,
                     int32_t* dx_exp, void* ws, hipStream_t stream)
{
    int8_t* wp = (int8_t*)ws;
    uint64_t* pmax = (uint64_t*)((char*)ws + align256((size_t)(g->R * g->S * t.Cp * t.Kp)));
    const int64_t npack = g->R * g->S * t.Cp * t.Kp;
    hipLaunchKernelGGL(k_tconv_pack, dim3(grid_for(npack, 256, 1024)), dim3(256), 0, stream, w, wp, (int32_t)g->K,
                       (int32_t)(g->R * g->S), (int32_t)g->C, t.Kp, t.Cp);
    int rc = launch_ok();
    if (rc) return rc;
    TconvArgs a{};
    a.dy = dy; a.wp = wp;
    a.N = (int32_t)g->N; a.H = (int32_t)g->H; a.W = (int32_t)g->W; a.C = (int32_t)g->C; a.K = (int32_t)g->K;
    a.Kp = t.Kp; a.Cp = t.Cp; a.P = (int32_t)P; a.Q = (int32_t)Q; a.R = (int32_t)g->R; a.S = (int32_t)g->S;
    a.sh = g->stride_h; a.sw = g->stride_w; a.ph = g->pad_h; a.pw = g->pad_w;
    a.tiles_h = t.tiles_h; a.tiles_w = t.tiles_w;
    conv_plan_set("phase");
    if (out_mode == ISEG_OUT_RAW) {
        a.out = (int32_t*)dx;
        if ((rc = launch_tconv_e<EPI_RAW>(t, a, stream))) return rc;
        hipLaunchKernelGGL(k_exp_sum, dim3(1), dim3(1), 0, stream, dx_exp, dy_exp, w_exp);
        return launch_ok();
    }
    a.pmax = pmax;
    a.npmax = t.gx * t.gy;
    if ((rc = launch_tconv_e<EPI_MAX>(t, a, stream))) return rc;
    a.out8 = (int8_t*)dx; a.exp_a = dy_exp; a.exp_b = w_exp; a.out_exp = dx_exp;
    return launch_tconv_e<EPI_Q8>(t, a, stream);
}

// A strided 1x1 conv (a projection shortcut): its dx is zero off the stride
// grid, and on it the stride-1 1x1 backward-data of dy over the P x Q output
// pixels.  That GEMM runs on the output grid (a quarter of the rows at stride
// 2, none of the products with the zeros between dy rows), and a pass writes
// dx with the zeros interleaved.  The zeros change neither the max nor any
// code, so the result and its exponent are those of the full backward-data.
static bool strided_1x1(const iseg_conv_geom* g)
{
    return g->R == 1 && g->S == 1 && g->pad_h == 0 && g->pad_w == 0 && (g->stride_h > 1 || g->stride_w > 1) &&
           g->C % 16 == 0 && g->N > 0;
}

static iseg_conv_geom strided_1x1_inner(const iseg_conv_geom* g, int64_t P, int64_t Q)
{
    iseg_conv_geom s = *g;
    s.H = P; s.W = Q; s.stride_h = 1; s.stride_w = 1; s.dil_h = 1; s.dil_w = 1;
    return s;
}

// dx from the output-grid result: 16-byte pieces of each pixel's row, the
// stride grid's pixels copied, all others zero
__global__ __launch_bounds__(256) void k_stride_scatter(const uint4* __restrict__ src, uint4* __restrict__ dst,
                                                        int64_t N, int32_t H, int32_t W, int32_t P, int32_t Q,
                                                        int32_t sh, int32_t sw, int32_t row16)
{
    const int64_t n16 = N * H * W * (int64_t)row16;
    const int64_t hw = (int64_t)H * W;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n16; i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t pix = i / row16;
        const int32_t k = (int32_t)(i - pix * row16);
        const int64_t n = pix / hw;
        const int32_t rem = (int32_t)(pix - n * hw);
        const int32_t h = rem / W, w = rem - h * W;
        uint4 v = make_uint4(0u, 0u, 0u, 0u);
        if (h % sh == 0 && w % sw == 0 && h / sh < P && w / sw < Q)
            v = src[((n * P + h / sh) * Q + w / sw) * row16 + k];
        dst[i] = v;
    }
}

static size_t conv_bwd_data_core_ws(const iseg_conv_geom* g, int32_t out_mode);

static size_t strided_1x1_ws(const iseg_conv_geom* g, int32_t out_mode, int64_t P, int64_t Q)
{
    const iseg_conv_geom s = strided_1x1_inner(g, P, Q);
    const size_t es = out_mode == ISEG_OUT_Q8 ? 1 : 4;
    return align256((size_t)(g->N * P * Q * g->C) * es) + conv_bwd_data_core_ws(&s, out_mode);
}

static size_t conv_bwd_data_core_ws(const iseg_conv_geom* g, int32_t out_mode)
{
    int64_t P, Q;
    if (!geom_ok(g, &P, &Q)) return 0;
    const size_t s1 = strided_1x1(g) ? strided_1x1_ws(g, out_mode, P, Q) : 0;
    const TconvPlan tp = tconv_plan(g);
    if (tp.ok) {
        const size_t st = 256 + tconv_ws_bytes(g, tp);
        return st > s1 ? st : s1;
    }
    size_t s = 256 + align256((size_t)(g->K * g->R * g->S * g->C));
    if (out_mode == ISEG_OUT_Q8) {
        size_t big = align256((size_t)(g->N * g->H * g->W * g->C) * 4);
        const size_t s16 = staged_ws_bytes(g->N * g->H * g->W, g->C);
        big = big > s16 ? big : s16;
        const DmaPlan dp = dma_plan(g->N * g->H * g->W, (int32_t)g->C, (int32_t)(g->K * g->R * g->S), true);
        const size_t sk = dma_split_bytes(dp, g->N * g->H * g->W, (int32_t)g->C);
        big = big > sk ? big : sk;
        const HaloPlan hp = halo_plan(g->N, g->H, g->W, g->K, g->C, (int)g->R, (int)g->S, g->stride_h,
                                      g->stride_w, g->dil_h, g->dil_w);
        if (hp.ok) {
            const size_t sh = halo_staged_ws_bytes(hp, g->N, g->H, g->W, g->C);
            big = big > sh ? big : sh;
        }
        s += big + conv_pmax_bytes(g->N * g->H * g->W, g->C, hp, g->N, g->H, g->W);
    }
    s += kpad_bytes(g);
    return s > s1 ? s : s1;
}

// backward-data with the transposed weights either built here from w (KRSC) or
// given by the caller (wt_in in layout wt_kind); a given layout that the
// chosen path does not use is ignored and the path builds its own
static int conv_bwd_data_core(const int8_t* dy, const int32_t* dy_exp, const int8_t* w, const int32_t* w_exp,
                              const int8_t* wt_in, int32_t wt_kind, const iseg_conv_geom* g, int32_t out_mode,
                              void* dx, int32_t* dx_exp, void* ws, size_t ws_bytes, int32_t* dev_status,
                              hipStream_t stream)
{
    (void)dev_status;
    int64_t P, Q;
    if (!geom_ok(g, &P, &Q)) return ISEG_ERR_SHAPE;
    if (out_mode != ISEG_OUT_Q8 && out_mode != ISEG_OUT_RAW) return ISEG_ERR_ARG;
    if (!dy_exp || !w_exp || !dx_exp || (g->N > 0 && (!dy || !w || !dx))) return ISEG_ERR_ARG;
    if (g->K * g->R * g->S > kMaxKred) return ISEG_ERR_UNSUPPORTED;
    if (!ws || ws_bytes < conv_bwd_data_core_ws(g, out_mode)) return ISEG_ERR_WORKSPACE;
    if (strided_1x1(g) && ((uintptr_t)dx & 15) == 0) {
        const iseg_conv_geom s = strided_1x1_inner(g, P, Q);
        const size_t es = out_mode == ISEG_OUT_Q8 ? 1 : 4;
        const size_t sub = align256((size_t)(g->N * P * Q * g->C) * es);
        int rc = conv_bwd_data_core(dy, dy_exp, w, w_exp, wt_in, wt_kind, &s, out_mode, ws, dx_exp,
                                    (char*)ws + sub, ws_bytes - sub, dev_status, stream);
        if (rc) return rc;
        conv_plan_set("strided_1x1");
        const int32_t row16 = (int32_t)(g->C * (int64_t)es / 16);
        hipLaunchKernelGGL(k_stride_scatter, dim3(grid_for(g->N * g->H * g->W * row16, 256, 8192)), dim3(256), 0,
                           stream, (const uint4*)ws, (uint4*)dx, g->N, (int32_t)g->H, (int32_t)g->W, (int32_t)P,
                           (int32_t)Q, g->stride_h, g->stride_w, row16);
        return launch_ok();
    }
    // ws: [max][transposed weights][per-block max partials][output staging]
    unsigned long long* maxp = (unsigned long long*)ws;
    const HaloPlan hp = halo_plan(g->N, g->H, g->W, g->K, g->C, (int)g->R, (int)g->S, g->stride_h, g->stride_w,
                                  g->dil_h, g->dil_w);
    int8_t* wt_ws = (int8_t*)ws + 256;
    const size_t wt_bytes = align256((size_t)(g->K * g->R * g->S * g->C));
    uint64_t* pmax = nullptr;
    int32_t* acc = (int32_t*)dx;
    if (out_mode == ISEG_OUT_Q8) {
        pmax = (uint64_t*)((char*)ws + 256 + wt_bytes);
        acc = (int32_t*)((char*)pmax + conv_pmax_bytes(g->N * g->H * g->W, g->C, hp, g->N, g->H, g->W));
    }
    int rc;
    // the caller's transposed weights when they are in the layout a path needs
    auto pick_wt = [&](int32_t kind) -> const int8_t* {
        return (wt_in && wt_kind == kind && ((uintptr_t)wt_in & 15) == 0) ? wt_in : wt_ws;
    };
    const int8_t* wt = wt_ws;
    const M32Plan mp = m32_plan(g->N, g->H, g->W, g->K, g->C, (int)g->R, (int)g->S, g->stride_h, g->stride_w,
                                g->dil_h, g->dil_w);
    wt = pick_wt(ISEG_WT_CRSK_FLIP);
    if (mp.ok && (((uintptr_t)dy | (uintptr_t)wt | (uintptr_t)dx) & 15) == 0) {
        conv_plan_set("m32");
        if (wt != wt_in && (rc = launch_w_transpose(w, wt_ws, g->K, g->R * g->S, g->C, true, stream))) return rc;
        HaloArgs h{};
        h.src = dy; h.wmat = wt; h.out = (int32_t*)dx;
        h.N = (int32_t)g->N; h.Hs = (int32_t)P; h.Ws = (int32_t)Q; h.Ci = (int32_t)g->K;
        h.Ho = (int32_t)g->H; h.Wo = (int32_t)g->W; h.Nout = (int32_t)g->C;
        h.ph = g->dil_h * (int32_t)(g->R - 1) - g->pad_h; h.pw = g->dil_w * (int32_t)(g->S - 1) - g->pad_w;
        h.dh = g->dil_h; h.dw = g->dil_w;
        if (out_mode == ISEG_OUT_RAW) {
            if ((rc = launch_m32(mp, h, EPI_RAW, ISEG_KID_CONV_BWD_DATA, stream))) return rc;
            hipLaunchKernelGGL(k_exp_sum, dim3(1), dim3(1), 0, stream, dx_exp, dy_exp, w_exp);
            return launch_ok();
        }
        return m32_q8(mp, h, ISEG_KID_CONV_BWD_DATA, dy_exp, w_exp, (int8_t*)dx, dx_exp, pmax, stream);
    }
    const PersistPlan pp = persist_plan(g->N, g->H, g->W, g->K, g->C, (int)g->R, (int)g->S, g->stride_h,
                                        g->stride_w, g->dil_h, g->dil_w);
    wt = pick_wt(ISEG_WT_CRSK_FLIP);
    if (pp.ok && (((uintptr_t)dy | (uintptr_t)wt | (uintptr_t)dx) & 15) == 0) {
        conv_plan_set("persist");
        // stride 1: dx = conv(dy, flipped W^T) with padding dil (R - 1) - pad
        if (wt != wt_in && (rc = launch_w_transpose(w, wt_ws, g->K, g->R * g->S, g->C, true, stream))) return rc;
        HaloArgs h{};
        h.src = dy; h.wmat = wt; h.out = (int32_t*)dx;
        h.N = (int32_t)g->N; h.Hs = (int32_t)P; h.Ws = (int32_t)Q; h.Ci = (int32_t)g->K;
        h.Ho = (int32_t)g->H; h.Wo = (int32_t)g->W; h.Nout = (int32_t)g->C;
        h.ph = g->dil_h * (int32_t)(g->R - 1) - g->pad_h; h.pw = g->dil_w * (int32_t)(g->S - 1) - g->pad_w;
        h.dh = g->dil_h; h.dw = g->dil_w;
        if (out_mode == ISEG_OUT_RAW) {
            if ((rc = launch_persist(pp, h, EPI_RAW, ISEG_KID_CONV_BWD_DATA, stream))) return rc;
            hipLaunchKernelGGL(k_exp_sum, dim3(1), dim3(1), 0, stream, dx_exp, dy_exp, w_exp);
            return launch_ok();
        }
        return persist_q8(pp, h, ISEG_KID_CONV_BWD_DATA, dy_exp, w_exp, (int8_t*)dx, dx_exp, pmax, stream);
    }
    wt = pick_wt(ISEG_WT_CRSK_FLIP);
    if (hp.ok && (((uintptr_t)dy | (uintptr_t)wt | (uintptr_t)dx | (uintptr_t)acc) & 15) == 0) {
        conv_plan_set("halo");
        // stride 1: dx = conv(dy, flipped W^T) with padding dil (R - 1) - pad
        if (wt != wt_in && (rc = launch_w_transpose(w, wt_ws, g->K, g->R * g->S, g->C, true, stream))) return rc;
        HaloArgs h{};
        h.src = dy; h.wmat = wt; h.out = acc;
        const int64_t rows = g->N * g->H * g->W;
        h.out16 = out_mode == ISEG_OUT_Q8 ? (int16_t*)acc : nullptr;
        h.tshift = (uint8_t*)acc + align256((size_t)(rows * g->C) * 2);
        h.N = (int32_t)g->N; h.Hs = (int32_t)P; h.Ws = (int32_t)Q; h.Ci = (int32_t)g->K;
        h.Ho = (int32_t)g->H; h.Wo = (int32_t)g->W; h.Nout = (int32_t)g->C;
        h.ph = g->dil_h * (int32_t)(g->R - 1) - g->pad_h; h.pw = g->dil_w * (int32_t)(g->S - 1) - g->pad_w;
        h.dh = g->dil_h; h.dw = g->dil_w;
        if (out_mode == ISEG_OUT_RAW) {
            if ((rc = launch_halo(hp, h, EPI_RAW, ISEG_KID_CONV_BWD_DATA, stream))) return rc;
            hipLaunchKernelGGL(k_exp_sum, dim3(1), dim3(1), 0, stream, dx_exp, dy_exp, w_exp);
            return launch_ok();
        }
        return halo_q8(hp, h, ISEG_KID_CONV_BWD_DATA, dy_exp, w_exp, (int8_t*)dx, dx_exp, maxp, pmax, rows,
                       stream);
    }
    const TconvPlan tp = tconv_plan(g);
    if (tp.ok)
        return tconv_run(tp, g, P, Q, dy, dy_exp, w, w_exp, out_mode, dx, dx_exp, (char*)ws + 256, stream);
    if (kpad_ok(g) && (((uintptr_t)dy | (uintptr_t)dx) & 15) == 0) {
        const int64_t Kp = kpad_to(g->K), M = g->N * g->H * g->W;
        int8_t* dyp = (int8_t*)ws + (conv_bwd_data_core_ws(g, out_mode) - kpad_bytes(g));
        int8_t* wtp = dyp + align256((size_t)(M * Kp));
        if ((rc = launch_pad(dy, dyp, M, g->K, Kp, stream))) return rc;
        hipLaunchKernelGGL(k_wt_pad_1x1, dim3(grid_for(g->C * Kp, 256, 1024)), dim3(256), 0, stream, w, wtp,
                           (int32_t)g->K, (int32_t)g->C, (int32_t)Kp);
        if ((rc = launch_ok())) return rc;
        IgemmArgs a{};
        a.src = dyp; a.wmat = wtp; a.out = acc; a.pmax = pmax;
        a.out16 = nullptr; a.tshift = nullptr;
        a.Mrows = M;
        a.Nout = (int32_t)g->C; a.Kred = (int32_t)Kp; a.Ci = (int32_t)Kp;
        a.Hs = (int32_t)P; a.Ws = (int32_t)Q; a.Ho = (int32_t)g->H; a.Wo = (int32_t)g->W;
        a.R = 1; a.S = 1; a.sh = 1; a.sw = 1; a.ph = 0; a.pw = 0; a.dh = 1; a.dw = 1;
        if (igemm_dma_ok(a))
            return igemm_dma_run<MODE_BWD>(a, out_mode, dy_exp, w_exp, dx, dx_exp, pmax, acc, stream);
    }
    wt = pick_wt(ISEG_WT_CRSK);
    if (wt != wt_in && (rc = launch_w_transpose(w, wt_ws, g->K, g->R * g->S, g->C, false, stream))) return rc;
    IgemmArgs a{};
    a.src = dy; a.wmat = wt; a.out = acc; a.pmax = pmax;
    a.out16 = nullptr; a.tshift = nullptr;
    a.Mrows = g->N * g->H * g->W;
    a.Nout = (int32_t)g->C; a.Kred = (int32_t)(g->K * g->R * g->S); a.Ci = (int32_t)g->K;
    a.Hs = (int32_t)P; a.Ws = (int32_t)Q; a.Ho = (int32_t)g->H; a.Wo = (int32_t)g->W;
    a.R = (int32_t)g->R; a.S = (int32_t)g->S;
    a.sh = g->stride_h; a.sw = g->stride_w; a.ph = g->pad_h; a.pw = g->pad_w;
    a.dh = g->dil_h; a.dw = g->dil_w;
    if (igemm_dma_ok(a) && ((uintptr_t)dx & 15) == 0)
        return igemm_dma_run<MODE_BWD>(a, out_mode, dy_exp, w_exp, dx, dx_exp, pmax, acc, stream);
    int64_t nblk = 0;
    conv_plan_set("igemm");
    if ((rc = launch_igemm<MODE_BWD>(a, stream, &nblk))) return rc;
    if (out_mode == ISEG_OUT_RAW) {
        hipLaunchKernelGGL(k_exp_sum, dim3(1), dim3(1), 0, stream, dx_exp, dy_exp, w_exp);
        return launch_ok();
    }
    return launch_requant_apply(acc, ISEG_I32, a.Mrows * a.Nout, dy_exp, w_exp, 0, 8, 0, 1,
                                0, 0, 0, ISEG_I8, dx, dx_exp, nullptr, stream, pmax, nblk);
}

// ---------------------------------------------------------------------------
// Reductions longer than the exact-int32 bound (C R S of a forward conv or
// K R S of a backward-data conv above kMaxKred, e.g. a 7x7 conv from 4096
// channels): the summed channels are cut into at most kMaxKredSplits chunks of
// a multiple of 16 channels, each chunk's conv writes its exact int32 sums
// (one contiguous copy of the chunk's operand columns ahead of it), and the
// quantizer adds the chunks in int64, so the codes are those of the exact
// total (|sum| < 127^2 * 8 * 131071 < 2^38).  Final codes only: raw int32 sums
// of such a reduction need not fit int32.
// ---------------------------------------------------------------------------
constexpr int kMaxKredSplits = 8;

struct KredSplit {
    int splits = 0;        // 0: the reduction cannot be split within the limits
    int64_t chunk = 0;     // channels per chunk (the last chunk may hold fewer)
};

static KredSplit kred_split(int64_t ch, int64_t RS)
{
    KredSplit ks;
    const int64_t cmax = (kMaxKred / RS) & ~(int64_t)15;
    if (cmax < 16) return ks;
    const int64_t n = ceil_div64(ch, cmax);
    if (n > kMaxKredSplits) return ks;
    ks.chunk = (ceil_div64(ch, n) + 15) & ~(int64_t)15;     // <= cmax
    ks.splits = (int)ceil_div64(ch, ks.chunk);
    return ks;
}

// dst[r][c] = src[r][c0 + c] (r < rows, c < cn): a column slice of a
// row-major [rows][cols] int8 matrix, 16 bytes per lane when all aligned
__global__ __launch_bounds__(256) void k_gather_cols(const int8_t* __restrict__ src, int64_t rows, int64_t cols,
                                                     int64_t c0, int64_t cn, int8_t* __restrict__ dst)
{
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t t0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (((cols | c0 | cn) & 15) == 0 && (((uintptr_t)src | (uintptr_t)dst) & 15) == 0) {
        const int64_t vpr = cn >> 4;
        for (int64_t i = t0; i < rows * vpr; i += stride) {
            const int64_t r = i / vpr, v = i - r * vpr;
            *(int4*)(dst + r * cn + v * 16) = *(const int4*)(src + r * cols + c0 + v * 16);
        }
        return;
    }
    for (int64_t i = t0; i < rows * cn; i += stride) {
        const int64_t r = i / cn, c = i - r * cn;
        dst[i] = src[r * cols + c0 + c];
    }
}

static int launch_gather_cols(const int8_t* src, int64_t rows, int64_t cols, int64_t c0, int64_t cn, int8_t* dst,
                              hipStream_t s)
{
    if (rows * cn == 0) return ISEG_OK;
    const int64_t work = (((cols | c0 | cn) & 15) == 0) ? rows * (cn >> 4) : rows * cn;
    hipLaunchKernelGGL(k_gather_cols, dim3(grid_for(work, 256, 4096)), dim3(256), 0, s, src, rows, cols, c0, cn, dst);
    return launch_ok();
}

// workspace: [max word][operand chunk][weight chunk (forward)][int32 sums of
// every chunk][max partials][the chunk convs' own workspace]
struct KredLayout {
    KredSplit ks;
    int64_t rows_a = 0, n = 0;
    size_t a_off = 0, w_off = 0, part_off = 0, pmax_off = 0, sub_off = 0, sub_bytes = 0, total = 0;
};

// The long reduction on the direct-to-LDS implicit GEMM when its shape
// allows (64-channel multiples, 16-byte aligned operands): the (tap, 64-channel
// chunk) steps are split over gridDim.z so that every split sums at most
// kMaxKred / 64 steps exactly in int32, with more splits (up to
// kMaxKredSplits) while the output tiles alone leave CUs idle; the int32
// partials go to the workspace and the quantizer adds them in int64.
// workspace: [max word][transposed weights (backward-data)][int32 partials of
// every split][max partials]
struct KredDma {
    bool ok = false;
    DmaPlan p{};
    size_t wt_off = 0, part_off = 0, pmax_off = 0, total = 0;
};

static KredDma kred_dma_plan(bool bwd, const iseg_conv_geom* g)
{
    KredDma d;
    int64_t P, Q;
    if (!geom_ok(g, &P, &Q)) return d;
    const int64_t Ci = bwd ? g->K : g->C, Nout = bwd ? g->C : g->K;
    const int64_t Mrows = bwd ? g->N * g->H * g->W : g->N * P * Q;
    if (Ci % 64 || Nout % 64 || g->R * g->S > 64 || Mrows < 1 || Mrows >= ((int64_t)1 << 31)) return d;
    const int64_t nk_full = g->R * g->S * (Ci / BK);
    int S = (int)ceil_div64(nk_full, kMaxKred / BK);
    if (S > kMaxKredSplits) return d;
    d.p.two_pass = false;
    d.p.bm = 128;
    d.p.bn = Nout % 128 == 0 ? 128 : 64;
    const int64_t blocks = ceil_div64(Mrows, d.p.bm) * (Nout / d.p.bn);
    while (S < kMaxKredSplits && blocks * S < ISEG_IGEMM_SPLIT_BLOCKS) S++;
    d.p.splits = S;
    size_t o = 256;
    d.wt_off = o;
    if (bwd) o += align256((size_t)(g->K * g->R * g->S * g->C));
    d.part_off = o;
    o += align256((size_t)(S * Mrows * Nout) * 4);
    d.pmax_off = o;
    o += align256(512 * 8);
    d.total = o;
    d.ok = true;
    return d;
}

static int conv_kred_dma(bool bwd, const KredDma& d, const int8_t* src, const int32_t* a_exp, const int8_t* w,
                         const int32_t* w_exp, const int8_t* wt_in, int32_t wt_kind, const iseg_conv_geom* g,
                         int8_t* out, int32_t* out_exp, void* ws, hipStream_t stream)
{
    int64_t P, Q;
    geom_ok(g, &P, &Q);
    char* base = (char*)ws;
    int32_t* part = (int32_t*)(base + d.part_off);
    uint64_t* pmax = (uint64_t*)(base + d.pmax_off);
    int rc;
    IgemmArgs a{};
    if (bwd) {
        int8_t* wt_ws = (int8_t*)(base + d.wt_off);
        const bool given = wt_in && wt_kind == ISEG_WT_CRSK && ((uintptr_t)wt_in & 15) == 0;
        if (!given && (rc = launch_w_transpose(w, wt_ws, g->K, g->R * g->S, g->C, false, stream))) return rc;
        a.src = src; a.wmat = given ? wt_in : wt_ws;
        a.Mrows = g->N * g->H * g->W;
        a.Nout = (int32_t)g->C; a.Kred = (int32_t)(g->K * g->R * g->S); a.Ci = (int32_t)g->K;
        a.Hs = (int32_t)P; a.Ws = (int32_t)Q; a.Ho = (int32_t)g->H; a.Wo = (int32_t)g->W;
    } else {
        a.src = src; a.wmat = w;
        a.Mrows = g->N * P * Q;
        a.Nout = (int32_t)g->K; a.Kred = (int32_t)(g->C * g->R * g->S); a.Ci = (int32_t)g->C;
        a.Hs = (int32_t)g->H; a.Ws = (int32_t)g->W; a.Ho = (int32_t)P; a.Wo = (int32_t)Q;
    }
    a.R = (int32_t)g->R; a.S = (int32_t)g->S;
    a.sh = g->stride_h; a.sw = g->stride_w; a.ph = g->pad_h; a.pw = g->pad_w;
    a.dh = g->dil_h; a.dw = g->dil_w;
    a.out = part; a.pmax = nullptr; a.out16 = nullptr; a.tshift = nullptr;
    if (!igemm_dma_ok(a)) return ISEG_ERR_UNSUPPORTED;
    a.tap_balance = (bwd ? every_tile_skips<MODE_BWD>(a, d.p.bm) : every_tile_skips<MODE_FWD>(a, d.p.bm)) ? 1 : 0;
    int64_t nblk = 0;
    rc = bwd ? launch_igemm_dma<MODE_BWD>(a, d.p, EPI_PART, stream, &nblk)
             : launch_igemm_dma<MODE_FWD>(a, d.p, EPI_PART, stream, &nblk);
    if (rc) return rc;
    conv_plan_set("kred_dma_split");
    const int64_t n = a.Mrows * a.Nout;
    int64_t npmax = 0;
    int qg = 0;
    if ((rc = launch_wgrad_reduce_qg(part, n, d.p.splits, nullptr, pmax, &npmax, stream, &qg))) return rc;
    if (qg != d.p.splits) return ISEG_ERR_UNSUPPORTED;     // splits <= 8 and n % 64 == 0 make it fuse
    return launch_requant_splits(part, d.p.splits, n, a_exp, w_exp, 8, 0, 1, 0, 0, 0, out, out_exp, stream, pmax,
                                 npmax);
}

static bool kred_dma_ready(bool bwd, const KredDma& d, const int8_t* src, const int8_t* w)
{
    return d.ok && (((uintptr_t)src | (uintptr_t)(bwd ? nullptr : w)) & 15) == 0;
}

static bool kred_layout(bool bwd, const iseg_conv_geom* g, KredLayout* L)
{
    int64_t P, Q;
    if (!geom_ok(g, &P, &Q)) return false;
    const int64_t ch = bwd ? g->K : g->C, RS = g->R * g->S;
    L->ks = kred_split(ch, RS);
    if (!L->ks.splits) return false;
    L->rows_a = bwd ? g->N * P * Q : g->N * g->H * g->W;
    L->n = bwd ? g->N * g->H * g->W * g->C : g->N * P * Q * g->K;
    if (L->n % 4) return false;
    size_t o = 256;
    L->a_off = o;
    o += align256((size_t)(L->rows_a * L->ks.chunk));
    L->w_off = o;
    if (!bwd) o += align256((size_t)(g->K * RS * L->ks.chunk));
    L->part_off = o;
    o += align256((size_t)(L->ks.splits * L->n) * 4);
    L->pmax_off = o;
    o += align256(512 * 8);
    size_t sub = 0;
    const int64_t last = ch - (int64_t)(L->ks.splits - 1) * L->ks.chunk;
    for (int64_t cn : {L->ks.chunk, last}) {
        iseg_conv_geom s = *g;
        (bwd ? s.K : s.C) = cn;
        const size_t b = bwd ? conv_bwd_data_core_ws(&s, ISEG_OUT_RAW) : conv_fwd_core_ws(&s, ISEG_OUT_RAW);
        sub = sub > b ? sub : b;
    }
    L->sub_off = o;
    L->sub_bytes = sub;
    L->total = o + sub;
    return true;
}

static size_t kred_ws(bool bwd, const iseg_conv_geom* g)
{
    KredLayout L;
    const size_t gs = kred_layout(bwd, g, &L) ? L.total : 0;
    const KredDma d = kred_dma_plan(bwd, g);
    const size_t ds = d.ok ? d.total : 0;
    return gs > ds ? gs : ds;
}

static int conv_kred_split(bool bwd, const int8_t* a, const int32_t* a_exp, const int8_t* w, const int32_t* w_exp,
                           const int8_t* wt_in, int32_t wt_kind, const iseg_conv_geom* g, int8_t* out,
                           int32_t* out_exp, void* ws, size_t ws_bytes, int32_t* dev_status, hipStream_t stream)
{
    KredLayout L;
    if (!kred_layout(bwd, g, &L)) return ISEG_ERR_UNSUPPORTED;
    if (!ws || ws_bytes < kred_ws(bwd, g)) return ISEG_ERR_WORKSPACE;
    const KredDma d = kred_dma_plan(bwd, g);
    if (kred_dma_ready(bwd, d, a, w))
        return conv_kred_dma(bwd, d, a, a_exp, w, w_exp, wt_in, wt_kind, g, out, out_exp, ws, stream);
    char* base = (char*)ws;
    int8_t* ac = (int8_t*)(base + L.a_off);
    int8_t* wc = (int8_t*)(base + L.w_off);
    int32_t* part = (int32_t*)(base + L.part_off);
    uint64_t* pmax = (uint64_t*)(base + L.pmax_off);
    void* sws = base + L.sub_off;
    const int64_t ch = bwd ? g->K : g->C, RS = g->R * g->S;
    int rc;
    conv_plan_set("kred_split");
    if (L.n == 0) {     // empty batch: the exponent of an all-zero tensor
        if ((rc = launch_fill_u32(base, 2, 0, stream))) return rc;
        return launch_requant_apply(part, ISEG_I32, 0, a_exp, w_exp, 0, 8, 0, 1, 0, 0, 0, ISEG_I8, out, out_exp,
                                    (const unsigned long long*)base, stream);
    }
    for (int i = 0; i < L.ks.splits; i++) {
        const int64_t c0 = (int64_t)i * L.ks.chunk;
        const int64_t cn = ch - c0 < L.ks.chunk ? ch - c0 : L.ks.chunk;
        iseg_conv_geom s = *g;
        int32_t* pi = part + (int64_t)i * L.n;
        if ((rc = launch_gather_cols(a, L.rows_a, ch, c0, cn, ac, stream))) return rc;
        if (bwd) {
            s.K = cn;
            rc = conv_bwd_data_core(ac, a_exp, w + c0 * RS * g->C, w_exp, nullptr, ISEG_WT_NONE, &s, ISEG_OUT_RAW,
                                    pi, out_exp, sws, L.sub_bytes, dev_status, stream);
        } else {
            s.C = cn;
            if ((rc = launch_gather_cols(w, g->K * RS, ch, c0, cn, wc, stream))) return rc;
            rc = conv_fwd_core(ac, a_exp, wc, w_exp, &s, ISEG_OUT_RAW, pi, out_exp, sws, L.sub_bytes, dev_status,
                               stream);
        }
        if (rc) return rc;
    }
    conv_plan_set("kred_split");
    int64_t npmax = 0;
    int qg = 0;
    if ((rc = launch_wgrad_reduce_qg(part, L.n, L.ks.splits, nullptr, pmax, &npmax, stream, &qg))) return rc;
    if (qg != L.ks.splits) return ISEG_ERR_UNSUPPORTED;     // splits <= 8 and n % 4 == 0 make it fuse
    return launch_requant_splits(part, L.ks.splits, L.n, a_exp, w_exp, 8, 0, 1, 0, 0, 0, out, out_exp, stream,
                                 pmax, npmax);
}

static bool conv_long_kred(bool bwd, const iseg_conv_geom* g)
{
    return (bwd ? g->K : g->C) * g->R * g->S > kMaxKred;
}

extern "C" size_t iseg_conv_fwd_ws(const iseg_conv_geom* g, int32_t out_mode)
{
    if (out_mode == ISEG_OUT_Q8 && g && conv_long_kred(false, g)) return kred_ws(false, g);
    return conv_fwd_core_ws(g, out_mode);
}

extern "C" int iseg_conv_fwd(const int8_t* x, const int32_t* x_exp, const int8_t* w, const int32_t* w_exp,
                             const iseg_conv_geom* g, int32_t out_mode, void* y, int32_t* y_exp,
                             void* ws, size_t ws_bytes, int32_t* dev_status, hipStream_t stream)
{
    ProfScope prof_scope(ISEG_KID_CONV_FWD, stream);
    conv_plan_set("none");
    int64_t P, Q;
    if (!g || !geom_ok(g, &P, &Q)) return ISEG_ERR_SHAPE;
    if (out_mode == ISEG_OUT_Q8 && conv_long_kred(false, g)) {
        if (!x_exp || !w_exp || !y_exp || (g->N > 0 && (!x || !w || !y))) return ISEG_ERR_ARG;
        return conv_kred_split(false, x, x_exp, w, w_exp, nullptr, ISEG_WT_NONE, g, (int8_t*)y, y_exp, ws, ws_bytes,
                               dev_status, stream);
    }
    return conv_fwd_core(x, x_exp, w, w_exp, g, out_mode, y, y_exp, ws, ws_bytes, dev_status, stream);
}

extern "C" size_t iseg_conv_bwd_data_ws(const iseg_conv_geom* g, int32_t out_mode)
{
    if (out_mode == ISEG_OUT_Q8 && g && conv_long_kred(true, g)) return kred_ws(true, g);
    return conv_bwd_data_core_ws(g, out_mode);
}

static int conv_bwd_data_impl(const int8_t* dy, const int32_t* dy_exp, const int8_t* w, const int32_t* w_exp,
                              const int8_t* wt_in, int32_t wt_kind, const iseg_conv_geom* g, int32_t out_mode,
                              void* dx, int32_t* dx_exp, void* ws, size_t ws_bytes, int32_t* dev_status,
                              hipStream_t stream)
{
    ProfScope prof_scope(ISEG_KID_CONV_BWD_DATA, stream);
    conv_plan_set("none");
    int64_t P, Q;
    if (!g || !geom_ok(g, &P, &Q)) return ISEG_ERR_SHAPE;
    if (out_mode == ISEG_OUT_Q8 && conv_long_kred(true, g)) {
        if (!dy_exp || !w_exp || !dx_exp || (g->N > 0 && (!dy || !w || !dx))) return ISEG_ERR_ARG;
        return conv_kred_split(true, dy, dy_exp, w, w_exp, wt_in, wt_kind, g, (int8_t*)dx, dx_exp, ws, ws_bytes,
                               dev_status, stream);
    }
    return conv_bwd_data_core(dy, dy_exp, w, w_exp, wt_in, wt_kind, g, out_mode, dx, dx_exp, ws, ws_bytes,
                              dev_status, stream);
}

extern "C" int iseg_conv_bwd_data(const int8_t* dy, const int32_t* dy_exp, const int8_t* w,
                                  const int32_t* w_exp, const iseg_conv_geom* g, int32_t out_mode,
                                  void* dx, int32_t* dx_exp, void* ws, size_t ws_bytes,
                                  int32_t* dev_status, hipStream_t stream)
{
    return conv_bwd_data_impl(dy, dy_exp, w, w_exp, nullptr, ISEG_WT_NONE, g, out_mode, dx, dx_exp, ws, ws_bytes,
                              dev_status, stream);
}

extern "C" int iseg_conv_bwd_data_t(const int8_t* dy, const int32_t* dy_exp, const int8_t* w,
                                    const int32_t* w_exp, const int8_t* wt, int32_t wt_kind,
                                    const iseg_conv_geom* g, int32_t out_mode, void* dx, int32_t* dx_exp,
                                    void* ws, size_t ws_bytes, int32_t* dev_status, hipStream_t stream)
{
    if (wt_kind != ISEG_WT_NONE && wt_kind != ISEG_WT_CRSK && wt_kind != ISEG_WT_CRSK_FLIP) return ISEG_ERR_ARG;
    return conv_bwd_data_impl(dy, dy_exp, w, w_exp, wt, wt_kind, g, out_mode, dx, dx_exp, ws, ws_bytes,
                              dev_status, stream);
}

extern "C" int32_t iseg_conv_bwd_data_wt_kind(const iseg_conv_geom* g)
{
    int64_t P, Q;
    if (!geom_ok(g, &P, &Q) || tconv_plan(g).ok) return ISEG_WT_NONE;
    if (conv_long_kred(true, g)) return kred_dma_plan(true, g).ok ? ISEG_WT_CRSK : ISEG_WT_NONE;
    const M32Plan mp = m32_plan(g->N, g->H, g->W, g->K, g->C, (int)g->R, (int)g->S, g->stride_h, g->stride_w,
                                g->dil_h, g->dil_w);
    const PersistPlan pp = persist_plan(g->N, g->H, g->W, g->K, g->C, (int)g->R, (int)g->S, g->stride_h,
                                        g->stride_w, g->dil_h, g->dil_w);
    const HaloPlan hp = halo_plan(g->N, g->H, g->W, g->K, g->C, (int)g->R, (int)g->S, g->stride_h, g->stride_w,
                                  g->dil_h, g->dil_w);
    return (mp.ok || pp.ok || hp.ok) ? ISEG_WT_CRSK_FLIP : ISEG_WT_CRSK;
}

extern "C" int iseg_weight_transpose_multi(const iseg_wt_desc* descs, int32_t n_desc, int64_t total_tiles,
                                           hipStream_t stream)
{
    if (n_desc == 0) return ISEG_OK;
    if (n_desc < 0 || total_tiles < 1 || !descs) return ISEG_ERR_ARG;
    if (total_tiles > ((int64_t)1 << 31) - 1) return ISEG_ERR_UNSUPPORTED;
    hipLaunchKernelGGL(k_w_transpose_multi, dim3((unsigned)total_tiles), dim3(256), 0, stream, descs, n_desc);
    return launch_ok();
}

// workspace: [max word][int64 sums][max partials][padded operands][int32
// split partials of the taps / split kernels][stem partials]
static size_t wgrad_part_region(int64_t NPQ, int64_t K, int64_t Cp, int64_t RS)
{
    const size_t t = wgrad_taps_part_bytes(NPQ, K, Cp, RS), r = wgrad_tr_part_bytes(NPQ, K, Cp, RS);
    return t > r ? t : r;
}

extern "C" size_t iseg_conv_bwd_weight_ws(const iseg_conv_geom* g, int32_t g_mode)
{
    int64_t P, Q;
    if (!geom_ok(g, &P, &Q)) return 0;
    (void)g_mode;
    const int64_t Cp = padded_c(g->C);
    const int64_t nwp = g->K * g->R * g->S * Cp;
    size_t s = 256 + align256((size_t)(g->K * g->R * g->S * g->C) * 8) + align256((size_t)wgrad_reduce_npmax(nwp) * 8);
    if (Cp != g->C)
        s += align256((size_t)(g->N * g->H * g->W * Cp)) + align256((size_t)nwp * 8);
    s += wgrad_part_region(g->N * P * Q, g->K, Cp, g->R * g->S);
    if (stem_kind(g->C, (int)g->R, (int)g->S, g->stride_h, g->stride_w, g->dil_h, g->dil_w, g->K)) {
        const int64_t nbx = g->N * ceil_div64(P, 16) * ceil_div64(Q, 32), nw = g->K * g->R * g->S * g->C;
        s += align256((size_t)(nbx * nw) * 4);
        const int nch = wgrad_reduce_chunks(nw, nbx);
        if (nch > 1) s += align256((size_t)(nch * nw) * 8);
    }
    return s;
}

extern "C" int iseg_conv_bwd_weight(const int8_t* dy, const int32_t* dy_exp, const int8_t* x,
                                    const int32_t* x_exp, const iseg_conv_geom* g, int32_t g_mode,
                                    int32_t bits, uint64_t seed, uint32_t tensor_id, uint32_t step,
                                    void* dw, int32_t* dw_exp, void* ws, size_t ws_bytes,
                                    int32_t* dev_status, hipStream_t stream)
{
    ProfScope prof_scope(ISEG_KID_CONV_WGRAD, stream);
    conv_plan_set("none");
    int64_t P, Q;
    if (!geom_ok(g, &P, &Q)) return ISEG_ERR_SHAPE;
    if (g_mode != ISEG_G_KEEP && g_mode != ISEG_G_DROP && g_mode != ISEG_G_RAW) return ISEG_ERR_ARG;
    if (g_mode != ISEG_G_RAW && (bits < 2 || bits > 8)) return ISEG_ERR_ARG;
    if (!dy_exp || !x_exp || !dw_exp || !dw || (g->N > 0 && (!dy || !x))) return ISEG_ERR_ARG;
    if (!ws || ws_bytes < iseg_conv_bwd_weight_ws(g, g_mode)) return ISEG_ERR_WORKSPACE;
    unsigned long long* maxp = (unsigned long long*)ws;
    const int64_t nw = g->K * g->R * g->S * g->C;
    const int64_t Cp = padded_c(g->C);
    const int64_t nwp = g->K * g->R * g->S * Cp;
    const int64_t NPQ = g->N * P * Q;
    const bool raw = g_mode == ISEG_G_RAW;
    const int keep = g_mode == ISEG_G_KEEP;
    char* wp = (char*)ws + 256;
    unsigned long long* acc = raw ? (unsigned long long*)dw : (unsigned long long*)wp;
    wp += align256((size_t)nw * 8);
    uint64_t* pmax = (uint64_t*)wp;
    wp += align256((size_t)wgrad_reduce_npmax(nwp) * 8);
    char* pad_region = wp;
    if (Cp != g->C) wp += align256((size_t)(g->N * g->H * g->W * Cp)) + align256((size_t)nwp * 8);
    int32_t* part = (int32_t*)wp;
    wp += wgrad_part_region(NPQ, g->K, Cp, g->R * g->S);
    int rc;
    int64_t npmax = 0;
    int qg = 0;                   // > 0: Q_G re-sums that many int32 splits (no int64 sums)
    // the int64 sums are done: their exponent (raw) or Q_G from the max partials
    auto finish = [&]() -> int {
        if (raw) {
            hipLaunchKernelGGL(k_exp_sum, dim3(1), dim3(1), 0, stream, dw_exp, dy_exp, x_exp);
            return launch_ok();
        }
        if (qg)
            return launch_requant_splits(part, qg, nw, keep ? dy_exp : nullptr, keep ? x_exp : nullptr, bits, 1, keep,
                                         seed, tensor_id, step, (int8_t*)dw, dw_exp, stream, pmax, npmax);
        return launch_requant_apply(acc, ISEG_I64, nw, keep ? dy_exp : nullptr, keep ? x_exp : nullptr, 0, bits, 1,
                                    keep, seed, tensor_id, step, ISEG_I8, dw, dw_exp, nullptr, stream, pmax, npmax);
    };
    const int stem = stem_kind(g->C, (int)g->R, (int)g->S, g->stride_h, g->stride_w, g->dil_h, g->dil_w, g->K);
    if (stem && g->N > 0 && ((uintptr_t)dy & 15) == 0) {
        conv_plan_set("wgrad_stem");
        // few-channel stem: MFMA over pixels, block partials, int64 sum + max partials
        int32_t* spart = (int32_t*)wp;
        HaloArgs h{};
        h.N = (int32_t)g->N; h.Hs = (int32_t)g->H; h.Ws = (int32_t)g->W; h.Ci = (int32_t)g->C;
        h.Ho = (int32_t)P; h.Wo = (int32_t)Q; h.Nout = (int32_t)g->K; h.ph = g->pad_h; h.pw = g->pad_w;
        h.tiles_y = (int)ceil_div64(P, 16); h.tiles_x = (int)ceil_div64(Q, 32);
        const unsigned nbx = (unsigned)(g->N * h.tiles_y * h.tiles_x);
        dim3 grid(nbx, (unsigned)(g->K / 64));
        if (stem == 1)
            ISEG_TIMED_LAUNCH(ISEG_KID_CONV_WGRAD, stream, (k_wgrad_stem<3, 3, 3, 1>), grid, dim3(256), 0, stream, dy,
                              x, spart, h);
        else
            ISEG_TIMED_LAUNCH(ISEG_KID_CONV_WGRAD, stream, (k_wgrad_stem<3, 7, 7, 2>), grid, dim3(256), 0, stream, dy,
                              x, spart, h);
        if ((rc = launch_ok())) return rc;
        if ((rc = launch_wgrad_reduce(spart, nw, nbx, (long long*)acc, raw ? nullptr : pmax, &npmax, stream)))
            return rc;
        return finish();
    }
    WgradArgs a{};
    a.dy = dy; a.x = x; a.acc = acc; a.part = nullptr;
    a.NPQ = NPQ; a.pix_per_split = 0;
    a.K = (int32_t)g->K; a.C = (int32_t)Cp; a.R = (int32_t)g->R; a.S = (int32_t)g->S;
    a.H = (int32_t)g->H; a.W = (int32_t)g->W; a.P = (int32_t)P; a.Q = (int32_t)Q;
    a.RSC = (int32_t)(g->R * g->S * Cp);
    a.sh = g->stride_h; a.sw = g->stride_w; a.ph = g->pad_h; a.pw = g->pad_w;
    a.dh = g->dil_h; a.dw = g->dil_w;
    if (Cp == g->C && wgrad_taps_shape(NPQ, g->K, Cp, g->R * g->S) && (((uintptr_t)x | (uintptr_t)dy) & 15) == 0 &&
        g->N * g->H * g->W * Cp < ((int64_t)1 << 31) && NPQ * g->K < ((int64_t)1 << 31)) {
        conv_plan_set("wgrad_taps");
        if ((rc = launch_wgrad_taps(a, part, raw ? nullptr : pmax, &npmax, stream, raw ? nullptr : &qg))) return rc;
        return finish();
    }
    if (Cp == g->C && wgrad_tr_ok(a)) {
        conv_plan_set("wgrad_tr");
        if ((rc = launch_wgrad_tr_split(a, part, raw ? nullptr : pmax, &npmax, stream, raw ? nullptr : &qg))) return rc;
        return finish();
    }
    // other shapes: atomic int64 accumulation (zero-filled), then the max pass
    conv_plan_set("wgrad_atomic");
    unsigned long long* accp = acc;
    if (Cp != g->C) {
        int8_t* xp = (int8_t*)pad_region;
        accp = (unsigned long long*)(pad_region + align256((size_t)(g->N * g->H * g->W * Cp)));
        if ((rc = launch_pad(x, xp, g->N * g->H * g->W, g->C, Cp, stream))) return rc;
        a.x = xp;
        a.acc = accp;
    }
    if ((rc = launch_fill_u32(accp, nwp * 2, 0, stream))) return rc;
    if ((rc = launch_wgrad(a, stream))) return rc;
    if (Cp != g->C) {
        hipLaunchKernelGGL(k_unpad_i64, dim3(grid_for(nw, 256, 4096)), dim3(256), 0, stream,
                           (const long long*)accp, (long long*)acc, g->K * g->R * g->S,
                           (int32_t)g->C, (int32_t)Cp);
        if ((rc = launch_ok())) return rc;
    }
    if (raw) return finish();
    if ((rc = launch_fill_u32(maxp, 2, 0, stream))) return rc;
    if ((rc = launch_absmax(acc, ISEG_I64, nw, maxp, dev_status, stream))) return rc;
    return launch_requant_apply(acc, ISEG_I64, nw, keep ? dy_exp : nullptr, keep ? x_exp : nullptr, 0, bits, 1, keep,
                                seed, tensor_id, step, ISEG_I8, dw, dw_exp, maxp, stream);
}
