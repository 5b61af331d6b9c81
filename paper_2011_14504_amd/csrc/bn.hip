// bn.hip -- L1 batch normalization (Eq. 12-15) and its backward on gfx950.
//
// Because the input of BN is an int8 code tensor, every per-element quantity
// of the forward (xhat_q, y, the ReLU mask, sgn(x - mu_q), the output code A)
// is a function of (channel, input code) only, and the backward's dx code is
// a function of (channel, sgn class, masked error code).  The work therefore
// splits into
//   * streaming passes over [M, C]: coalesced dword loads (four channels per
//     lane), four rows in flight per lane, per-channel sums reduced in LDS and
//     written as one partial per block and channel (no global atomics, so no
//     same-address serialization across blocks);
//   * finalize steps that reduce the partials and do the exact rational
//     arithmetic in __int128 once per channel or per table entry.  The
//     per-channel step runs in the tail of a streaming pass, in the last
//     block of each channel slice to finish (an arrival counter picks it, no
//     block waits), and grid-wide maxima in the last slice to finish; the
//     per-(channel, code) tables take one block per channel.
// sgn(x - mu_q) and the ReLU mask are monotone in the input code, so the
// streaming passes get them from two thresholds per channel instead of a
// table.
//
// Forward:  stats1 (block partials of sum q, min q, max q) -> stats2 (each
//           block first forms n_mu and the occupied code range of its slice
//           from them; sum |x - mu_q| | tails: n_sigma, den, the slice's
//           bound on b) -> fin2 (b; xhat codes, y, thresholds, max|y|, y
//           staged at each channel's own Q_A shift) -> apply (Q_A's shift from
//           the channels' maxima; A codes; table gather).
// Backward: exact E2 (k_E2 >= 15): stats (block partials of sum delta, sum
//           delta*xhat, sum sgn and the per-class extremes of delta) ->
//           per-channel kernel (dgamma, dbeta, the channel's bound on E1's
//           exponent, its dx values staged at that bound) -> apply (E1's
//           exponent from the channels' bounds; staged values rounded into
//           the gather table).  k_E2 < 15 adds a second streaming pass: stats
//           tails give each slice's max|gamma delta| (E2's scale is the
//           largest), stats2 sums the rounded E2 terms and its tails give the
//           slices' bounds on E1's exponent; a table kernel, then apply.
#include <mutex>
#include <type_traits>

#include "iseg_common.h"

namespace {

constexpr int kSentinelLo = -(1 << 30);
typedef short short2v __attribute__((ext_vector_type(2)));

// launch geometry of the streaming passes (compile-time tuning knobs)
#ifndef ISEG_BN_NT
#define ISEG_BN_NT 1024          // threads per streaming block
#endif
#ifndef ISEG_BN_BLOCKS
#define ISEG_BN_BLOCKS 256       // streaming blocks per call, all channel slices
#endif
#ifndef ISEG_BNF_STATS_CPL
#define ISEG_BNF_STATS_CPL 4     // channels per lane of the forward statistics
#endif
#ifndef ISEG_BNB_ROWS
#define ISEG_BNB_ROWS 2          // row groups per lane that size the backward statistics grid
#endif
constexpr int kMaxBlocks = ISEG_BN_BLOCKS;

// ---------------------------------------------------------------------------
// saved-state layout (documented in iseg.h)
// ---------------------------------------------------------------------------
struct Saved {
    int32_t* hdr;
    int32_t *n_mu, *n_sigma, *den, *qmin, *qmax;
    int32_t *t0, *p0, *mlo, *mhi;   // sgn/mask thresholds
    int16_t* xcode;                  // [C][256]
    uint8_t* flags;                  // [C][256]
    int8_t* acode;                   // [C][256]
    uint32_t* btab;                  // [C][256] by q & 0xff: y > 0, sgn, |sgn|, xhat code
    int16_t* ystg;                   // [C][256] ReLU(y) >> t_c (the output pass's staged A values)
};

size_t saved_bytes(int64_t C)
{
    return 256 + 9 * align256((size_t)C * 4) + align256((size_t)C * 512) +
           2 * align256((size_t)C * 256) + align256((size_t)C * 1024) + align256((size_t)C * 512);
}

Saved saved_map(void* base, int64_t C)
{
    char* p = (char*)base;
    Saved s;
    size_t v = align256((size_t)C * 4);
    s.hdr = (int32_t*)p; p += 256;
    s.n_mu = (int32_t*)p; p += v;
    s.n_sigma = (int32_t*)p; p += v;
    s.den = (int32_t*)p; p += v;
    s.qmin = (int32_t*)p; p += v;
    s.qmax = (int32_t*)p; p += v;
    s.t0 = (int32_t*)p; p += v;
    s.p0 = (int32_t*)p; p += v;
    s.mlo = (int32_t*)p; p += v;
    s.mhi = (int32_t*)p; p += v;
    s.xcode = (int16_t*)p; p += align256((size_t)C * 512);
    s.flags = (uint8_t*)p; p += align256((size_t)C * 256);
    s.acode = (int8_t*)p; p += align256((size_t)C * 256);
    s.btab = (uint32_t*)p; p += align256((size_t)C * 1024);
    s.ystg = (int16_t*)p;
    return s;
}

// ---------------------------------------------------------------------------
// streaming geometry: a block covers one channel slice of CS channels (CS % 4
// == 0, CS divides C); lane g of a row handles channels 4g..4g+3 of the slice;
// rpi rows are in flight per block step.
// ---------------------------------------------------------------------------
struct Stream {
    int64_t M;
    int32_t C, CS, G, rpi, gx;
};

int pick_cs(int64_t C, int csmax)
{
    for (int cs = csmax; cs >= 4; cs -= 4)
        if (C % cs == 0) return cs;
    return 0;
}

constexpr int kNT = ISEG_BN_NT;
constexpr int kWaves = kNT / 64;       // waves per streaming block

Stream make_stream(int64_t M, int64_t C, int cs, int cpl, int unroll, int max_blocks)
{
    Stream s;
    s.M = M; s.C = (int32_t)C; s.CS = cs; s.G = cs / cpl; s.rpi = kNT / s.G;
    int nsl = (int)(C / cs);
    int64_t want = max_blocks / nsl;
    if (want < 1) want = 1;
    int64_t rows = ceil_div64(M, (int64_t)s.rpi * unroll);
    s.gx = (int32_t)(rows < want ? rows : want);
    if (s.gx < 1) s.gx = 1;
    return s;
}

dim3 stream_grid(const Stream& s) { return dim3((unsigned)s.gx, (unsigned)(s.C / s.CS)); }

__device__ __forceinline__ bool stream_lane(const Stream& st, int& g, int& rsub)
{
    g = threadIdx.x % st.G;
    rsub = threadIdx.x / st.G;
    return rsub < st.rpi;
}

// Iterate the rows of this lane with U rows in flight; a lane covers CPL
// channels (4: one dword, 16: one 16-byte vector).  f(row, words[CPL/4]).
template <int CPL>
struct Vec { uint32_t w[CPL / 4]; };

template <int CPL>
__device__ __forceinline__ Vec<CPL> vload(const int8_t* p)
{
    Vec<CPL> v;
    if (CPL == 16) {
        uint4 t = *(const uint4*)p;
        v.w[0] = t.x; v.w[CPL / 4 > 1 ? 1 : 0] = t.y;
        if (CPL == 16) { v.w[2 % (CPL / 4)] = t.z; v.w[3 % (CPL / 4)] = t.w; }
    } else {
        v.w[0] = *(const uint32_t*)p;
    }
    return v;
}

template <int CPL>
__device__ __forceinline__ void vstore(int8_t* p, const Vec<CPL>& v)
{
    if (CPL == 16) *(uint4*)p = make_uint4(v.w[0], v.w[1 % (CPL / 4)], v.w[2 % (CPL / 4)], v.w[3 % (CPL / 4)]);
    else *(uint32_t*)p = v.w[0];
}

template <int CPL, int U, typename F>
__device__ __forceinline__ void stream_rows(const Stream& st, const int8_t* __restrict__ a, int c0,
                                            int rsub, F f)
{
    const int64_t step = (int64_t)gridDim.x * st.rpi;
    for (int64_t r = (int64_t)blockIdx.x * st.rpi + rsub; r < st.M; r += step * U) {
        Vec<CPL> v[U];
#pragma unroll
        for (int u = 0; u < U; u++) {
            int64_t rr = r + u * step;
            if (rr < st.M) v[u] = vload<CPL>(a + rr * st.C + c0);
        }
#pragma unroll
        for (int u = 0; u < U; u++) {
            int64_t rr = r + u * step;
            if (rr < st.M) f(rr, v[u]);
        }
    }
}

// two-input variant
template <int CPL, int U, typename F>
__device__ __forceinline__ void stream_rows2(const Stream& st, const int8_t* __restrict__ a,
                                             const int8_t* __restrict__ b, int c0, int rsub, F f)
{
    const int64_t step = (int64_t)gridDim.x * st.rpi;
    for (int64_t r = (int64_t)blockIdx.x * st.rpi + rsub; r < st.M; r += step * U) {
        Vec<CPL> va[U], vb[U];
#pragma unroll
        for (int u = 0; u < U; u++) {
            int64_t rr = r + u * step;
            if (rr < st.M) {
                va[u] = vload<CPL>(a + rr * st.C + c0);
                vb[u] = vload<CPL>(b + rr * st.C + c0);
            }
        }
#pragma unroll
        for (int u = 0; u < U; u++) {
            int64_t rr = r + u * step;
            if (rr < st.M) f(rr, va[u], vb[u]);
        }
    }
}

__device__ __forceinline__ int sbyte(uint32_t w, int i) { return (int)(int8_t)(w >> (8 * i)); }

__device__ __forceinline__ bool sx_ok(int32_t s_x) { return s_x >= -40 && s_x <= 16; }

// D = (x - mu_q) / 2^g for code q; g = min(s_x, e_mu)
__device__ __forceinline__ int64_t bn_D(int q, int32_t s_x, int32_t n_mu, int e_mu)
{
    int g = s_x < e_mu ? s_x : e_mu;
    return (int64_t)q * ((int64_t)1 << (s_x - g)) - (int64_t)n_mu * ((int64_t)1 << (e_mu - g));
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

// block-wide reduction of one value per thread (256 threads): xor-shuffles
// within each wave, then the four wave results through LDS (two barriers)
template <typename T, typename Op>
__device__ __forceinline__ T block_reduce(T v, Op op, T* sh)
{
    for (int o = 32; o > 0; o >>= 1) v = op(v, (T)__shfl_xor(v, o, 64));
    if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = v;
    __syncthreads();
    T r = sh[0];
    for (int k = 1; k < (int)(blockDim.x >> 6); k++) r = op(r, sh[k]);
    __syncthreads();
    return r;
}

struct OpAdd { template <typename T> __device__ T operator()(T a, T b) const { return a + b; } };
struct OpMin { template <typename T> __device__ T operator()(T a, T b) const { return a < b ? a : b; } };
struct OpMax { template <typename T> __device__ T operator()(T a, T b) const { return a > b ? a : b; } };

// v op v[lane ^ O]: for O = 16 or 32 with gfx950's cross-row swaps (VALU, no
// LDS traffic): v_permlane16_swap / v_permlane32_swap with both operands v
// leave v and its partner's value in the two results (which is which depends
// on the lane, so only commutative ops are folded); other O: an xor-shuffle.
template <int O>
__device__ __forceinline__ uint32_t lane_x32(uint32_t v, uint32_t* partner)
{
    if constexpr (O == 16) {
        const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
        *partner = r[1];
        return r[0];
    } else {
        const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
        *partner = r[1];
        return r[0];
    }
}

template <int O, typename T, typename Op>
__device__ __forceinline__ T xor_fold(T v, Op op)
{
    if constexpr (O != 16 && O != 32) {
        return op(v, (T)__shfl_xor(v, O, 64));
    } else if constexpr (sizeof(T) == 8) {
        const uint64_t u = (uint64_t)v;
        uint32_t lp, hp;
        const uint32_t la = lane_x32<O>((uint32_t)u, &lp);
        const uint32_t ha = lane_x32<O>((uint32_t)(u >> 32), &hp);
        return op((T)((uint64_t)la | ((uint64_t)ha << 32)), (T)((uint64_t)lp | ((uint64_t)hp << 32)));
    } else {
        uint32_t p;
        const uint32_t a = lane_x32<O>((uint32_t)v, &p);
        return op((T)a, (T)p);
    }
}

// Lanes of a wave that hold the same channels are G apart (G a power of two
// dividing 64): fold them so that every lane holds the total over the wave's
// lanes of its channels (straight-line code for a compile-time G; G = 0 or 64:
// nothing to fold).  Every lane of the wave must be active.
template <int G, typename T, typename Op>
__device__ __forceinline__ T fold_g(T v, Op op)
{
    if constexpr (G >= 1 && G < 64) return fold_g<2 * G>(xor_fold<G>(v, op), op);
    else return v;
}

// f(std::integral_constant<int, G>) for a slice whose row has G lanes: G
// itself when it is a power of two up to 64 (compile-time folds), else 0.
template <typename F>
__device__ __forceinline__ void with_g(int G, F f)
{
    switch (G) {
    case 1: f(std::integral_constant<int, 1>()); break;
    case 2: f(std::integral_constant<int, 2>()); break;
    case 4: f(std::integral_constant<int, 4>()); break;
    case 8: f(std::integral_constant<int, 8>()); break;
    case 16: f(std::integral_constant<int, 16>()); break;
    case 32: f(std::integral_constant<int, 32>()); break;
    case 64: f(std::integral_constant<int, 64>()); break;
    default: f(std::integral_constant<int, 0>()); break;
    }
}

__device__ __forceinline__ bool group_leader(int G)
{
    return ((G & (G - 1)) != 0 || G > 64) || (int)(threadIdx.x & 63) < G;
}

// Copy n 16-byte pieces (n <= V * kNT) from global memory into LDS, every load
// of a thread issued before its first store.
template <int V>
__device__ __forceinline__ void copy_to_lds(uint4* dst, const uint4* __restrict__ src, int n)
{
    uint4 v[V];
#pragma unroll
    for (int k = 0; k < V; k++) {
        const int i = threadIdx.x + k * kNT;
        if (i < n) v[k] = src[i];
    }
#pragma unroll
    for (int k = 0; k < V; k++) {
        const int i = threadIdx.x + k * kNT;
        if (i < n) dst[i] = v[k];
    }
}

// LDS tables are kept one dword longer per row than in global memory: a
// table row is 256 entries (a multiple of the bank count), so without the skew
// every channel's entry for the same input code would sit in the same bank,
// and real activations concentrate on a few codes.
constexpr int kRowB = 256 + 4;      // bytes per row of a byte table in LDS
constexpr int kRowW = 256 + 1;      // dwords per row of a dword table in LDS

// Copy `rows` rows of 256 bytes (global, contiguous) into LDS rows of kRowB
// bytes; every load of a thread is issued before its first store.
template <int V>
__device__ __forceinline__ void copy_rows_to_lds(int8_t* dst, const int8_t* __restrict__ src, int rows)
{
    const int n = rows * 16;
    uint4 v[V];
#pragma unroll
    for (int k = 0; k < V; k++) {
        const int i = threadIdx.x + k * kNT;
        if (i < n) v[k] = ((const uint4*)src)[i];
    }
#pragma unroll
    for (int k = 0; k < V; k++) {
        const int i = threadIdx.x + k * kNT;
        if (i < n) {
            uint32_t* d = (uint32_t*)(dst + (i >> 4) * kRowB + (i & 15) * 16);
            d[0] = v[k].x; d[1] = v[k].y; d[2] = v[k].z; d[3] = v[k].w;
        }
    }
}

// ---------------------------------------------------------------------------
// arrival counters.  The backward workspace starts with ctr_bytes(C) bytes of
// uint32 counters: ctr[0] counts the channel slices whose partials are final,
// ctr[1 + y] the blocks of slice y that have published theirs.  atomicInc
// with limit n - 1 hands n - 1 to the n-th arrival and wraps the counter to
// zero there, so each kernel leaves the counters as it found them (zero); no
// block ever waits for another.
// ---------------------------------------------------------------------------
size_t ctr_bytes(int64_t C) { return ISEG_BN_WS_ZERO(C); }   // >= 4 (1 + C / 4)

// Values that cross blocks inside one kernel (partials, per-channel results
// a later tail reads) are stored and loaded as relaxed agent-scope atomics:
// write-through stores and loads that are coherent across the XCDs' L2
// caches.  Device-scope fences would give the same ordering by writing back
// and invalidating each whole L2, far too costly once per block.
template <typename T>
__device__ __forceinline__ void st_x(T* p, T v) { __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }
template <typename T>
__device__ __forceinline__ T ld_x(const T* p) { return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }

// Called by every thread of a block after its st_x stores: true in all
// threads of the block that arrives last of n.  Each thread waits for its
// stores to complete (vmcnt 0) before the barrier, and the counter update
// follows the barrier, so every earlier arrival's stores precede the last
// block's ld_x loads.
__device__ __forceinline__ bool arrive_last(uint32_t* ctr, unsigned n)
{
    __shared__ int s_last;
    __builtin_amdgcn_s_waitcnt(0x0F70);     // vmcnt(0)
    __syncthreads();
    if (threadIdx.x == 0) s_last = atomicInc(ctr, n - 1) == n - 1;
    __syncthreads();
    return s_last != 0;
}

// max over the kNT threads of a block (every thread gets it)
template <typename T>
__device__ __forceinline__ T block_max_nt(T v, T* sh)
{
    for (int o = 32; o > 0; o >>= 1) { const T u = __shfl_xor(v, o, 64); v = u > v ? u : v; }
    if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = v;
    __syncthreads();
    T m = sh[0];
    for (int k = 1; k < kNT / 64; k++) m = sh[k] > m ? sh[k] : m;
    __syncthreads();
    return m;
}

// ---------------------------------------------------------------------------
// forward workspace.  It starts, like the backward's, with ctr_bytes(C)
// bytes of arrival counters that each call leaves at zero.
// ---------------------------------------------------------------------------
struct FwdWs {
    uint32_t* ctr;                   // arrival counters
    int32_t* b_glob;                 // exponent of Q_xhat's scale (fin2, block 0)
    int32_t *p_s1, *p_mm;            // [slice][gx][CS] partials: sum q; (min q + 128) | (max q + 128) << 16
    long long* p_abs;                // [gx][C]
    int32_t* sbmax;                  // [slices] largest channel bound on b of each slice (stats2's tails)
    unsigned long long* maxYc;       // [C] max |ReLU(y)| of channel c over its occupied codes (fin2)
};

size_t fwd_ws_bytes(const Stream& st)
{
    size_t pc = (size_t)st.gx * st.C;
    return ctr_bytes(st.C) + 256 + 2 * align256(pc * 4) + align256(pc * 8) + align256((size_t)st.C) +
           align256((size_t)st.C * 8);
}

FwdWs fwd_ws_map(void* base, const Stream& st)
{
    char* p = (char*)base;
    size_t pc = (size_t)st.gx * st.C;
    FwdWs w;
    w.ctr = (uint32_t*)p; p += ctr_bytes(st.C);
    w.b_glob = (int32_t*)p;
    p += 256;
    w.p_s1 = (int32_t*)p; p += align256(pc * 4);
    w.p_mm = (int32_t*)p; p += align256(pc * 4);
    w.p_abs = (long long*)p; p += align256(pc * 8);
    w.sbmax = (int32_t*)p; p += align256((size_t)st.C);       // slices <= C / 4
    w.maxYc = (unsigned long long*)p;
    return w;
}

// ---------------------------------------------------------------------------
// forward kernels
//
// stats1 | block partials of sum q, min q, max q
// stats2 | prologue: n_mu and the occupied code range of the slice's channels
//          from stats1's partials | tails: n_sigma, the denominator and each
//          channel's bound on max|xhat|; the slice's largest bound
// fin2   (one block per channel, one thread per code): b (Q_xhat's scale) from
//          the slices' bounds; xhat codes, y, sgn / ReLU thresholds, the
//          backward's entries, the channel's max|ReLU(y)| and ReLU(y) staged
//          at the channel's own Q_A shift
// apply  Q_A's shift r from the channels' maxima; the saved A codes; the
//          gather table from the staged values; table gather
// ---------------------------------------------------------------------------

// Partial rows of a slice tail in flight per thread: the thread of channel
// t % CS in row group t / CS reduces partial rows t / CS + k ng (ng = kNT /
// CS), kTailU of them per batch, all loads of a batch issued before the first
// is used (an index past the last row re-reads the group's first row, whose
// value the reduction ignores).
constexpr int kTailU = 8;

template <int CPL>
__global__ __launch_bounds__(1024) void k_bnf_stats1(const int8_t* __restrict__ x, Stream st, FwdWs w)
{
    __shared__ int32_t sS[128], sMin[128], sMax[128];
    __shared__ int32_t wst[3 * kWaves * 128];      // wave totals [quantity][wave][channel]
    const bool fold = (st.G & (st.G - 1)) == 0 && st.G <= 64;
    if (!fold && (int)threadIdx.x < st.CS) { sS[threadIdx.x] = 0; sMin[threadIdx.x] = 1000; sMax[threadIdx.x] = -1000; }
    __syncthreads();
    int g, rsub;
    const bool active = stream_lane(st, g, rsub);
    int s[CPL], mn[CPL], mx[CPL];
#pragma unroll
    for (int i = 0; i < CPL; i++) { s[i] = 0; mn[i] = 1000; mx[i] = -1000; }
    if (active) {
        int c0 = blockIdx.y * st.CS + g * CPL;
        stream_rows<CPL, 4>(st, x, c0, rsub, [&](int64_t, const Vec<CPL>& v) {
#pragma unroll
            for (int i = 0; i < CPL; i++) {
                int q = sbyte(v.w[i >> 2], i & 3);
                s[i] += q;
                mn[i] = q < mn[i] ? q : mn[i];
                mx[i] = q > mx[i] ? q : mx[i];
            }
        });
    }
    with_g(st.G, [&](auto gc) {
        constexpr int GG = decltype(gc)::value;
#pragma unroll
        for (int i = 0; i < CPL; i++) {
            s[i] = fold_g<GG>(s[i], OpAdd());
            mn[i] = fold_g<GG>(mn[i], OpMin());
            mx[i] = fold_g<GG>(mx[i], OpMax());
        }
    });
    // block totals: the 16 wave totals of each channel staged in LDS and summed
    // by one thread per channel (see k_bnb_stats); other widths: LDS atomics
    if (fold) {
        const int wv = threadIdx.x >> 6;
        if ((int)(threadIdx.x & 63) < st.G) {
#pragma unroll
            for (int i = 0; i < CPL; i++) {
                const int c = g * CPL + i;
                wst[wv * 128 + c] = s[i];
                wst[(kWaves + wv) * 128 + c] = mn[i];
                wst[(2 * kWaves + wv) * 128 + c] = mx[i];
            }
        }
        __syncthreads();
        if ((int)threadIdx.x < st.CS) {
            const int c = threadIdx.x;
            int bs = 0, bmn = 1000, bmx = -1000;
#pragma unroll 4
            for (int v = 0; v < kWaves; v++) {
                bs += wst[v * 128 + c];
                bmn = min(bmn, wst[(kWaves + v) * 128 + c]);
                bmx = max(bmx, wst[(2 * kWaves + v) * 128 + c]);
            }
            sS[c] = bs; sMin[c] = bmn; sMax[c] = bmx;
        }
    } else if (active && group_leader(st.G)) {
#pragma unroll
        for (int i = 0; i < CPL; i++) {
            atomicAdd(&sS[g * CPL + i], s[i]);
            atomicMin(&sMin[g * CPL + i], mn[i]);
            atomicMax(&sMax[g * CPL + i], mx[i]);
        }
    }
    __syncthreads();
    // every block holds at least one row of the slice, so its extremes are
    // codes; one contiguous row of partials per block, reduced by every block
    // of the next pass for its slice
    if ((int)threadIdx.x < st.CS) {
        const int64_t o = ((int64_t)blockIdx.y * st.gx + blockIdx.x) * st.CS + threadIdx.x;
        w.p_s1[o] = sS[threadIdx.x];
        w.p_mm[o] = (sMin[threadIdx.x] + 128) | ((sMax[threadIdx.x] + 128) << 16);
    }
}

// y on the grid 2^e_y of a channel's code q (before ReLU), and x-hat's code
struct FwdExps {
    int e_mu, e_sig, gg, e_g, e_b, e_xh, e_y, kx;
};

__device__ __forceinline__ FwdExps fwd_exps(int32_t s_x, int b, const BnCfg& cf)
{
    FwdExps e;
    e.e_mu = 2 - cf.k_mu; e.e_sig = 2 - cf.k_sigma;
    e.gg = s_x < e.e_mu ? s_x : e.e_mu;
    e.e_g = 2 - cf.k_gamma; e.e_b = 2 - cf.k_beta;
    e.kx = cf.k_xhat;
    e.e_xh = b - (cf.k_xhat - 1);
    e.e_y = (e.e_g + e.e_xh) < e.e_b ? (e.e_g + e.e_xh) : e.e_b;
    return e;
}

__device__ __forceinline__ i128 fwd_xcode(int64_t D, int32_t den, int b, const FwdExps& e)
{
    return clamp_k128(rhu128((i128)D, e.gg - e.e_sig + (e.kx - 1) - b, (i128)den), e.kx);
}

__device__ __forceinline__ i128 fwd_y(i128 nx, int gq, int bq, const FwdExps& e)
{
    return (i128)gq * nx * pow2_128(e.e_g + e.e_xh - e.e_y) + (i128)bq * pow2_128(e.e_b - e.e_y);
}

template <int CPL>
__global__ __launch_bounds__(1024) void k_bnf_stats2(const int8_t* __restrict__ x, const int32_t* x_exp,
                                                    Stream st, FwdWs w, Saved sv, BnCfg cf, int32_t* dev_status)
{
    __shared__ int32_t sSg[128], sNg[128];         // block sums of q and counts above each channel's T
    __shared__ long long tA[kNT];
    __shared__ int32_t rb[kNT / 64];
    __shared__ int32_t wst[2 * kWaves * 128];      // wave totals [quantity][wave][channel]
    const bool fold = (st.G & (st.G - 1)) == 0 && st.G <= 64;
    int32_t s_x = *x_exp;
    if (!sx_ok(s_x)) {
        if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) set_status(dev_status, ISEG_DEV_RANGE);
        s_x = -14;     // keep shifts defined; outputs are unspecified
    }
    if (!fold && (int)threadIdx.x < st.CS) { sSg[threadIdx.x] = 0; sNg[threadIdx.x] = 0; }
    // prologue: n_mu (Eq. 12) and the occupied code range of the slice's
    // channels from stats1's partial rows (every block of the slice forms them;
    // the slice's last block stores them)
    __shared__ int32_t sNmu[128], sLo[128], sHi[128];
    __shared__ long long sSum[128];
    {
        const int CS = st.CS, ng = kNT / CS, t = threadIdx.x, ch = t % CS, grp = t / CS;
        const int32_t* ps = w.p_s1 + (int64_t)blockIdx.y * st.gx * CS;
        const int32_t* pm = w.p_mm + (int64_t)blockIdx.y * st.gx * CS;
        long long sum = 0;
        int lo = 255, hi = 0;
        if (grp < ng)
            for (int b0 = grp; b0 < st.gx; b0 += kTailU * ng) {
                int32_t vs[kTailU], vm[kTailU];
#pragma unroll
                for (int u = 0; u < kTailU; u++) {
                    const int b = b0 + u * ng;
                    const int64_t q = (int64_t)(b < st.gx ? b : b0) * CS + ch;
                    vs[u] = ps[q];
                    vm[u] = pm[q];
                }
#pragma unroll
                for (int u = 0; u < kTailU; u++) {
                    if (b0 + u * ng < st.gx) sum += vs[u];
                    lo = min(lo, vm[u] & 0xffff);       // a repeated row changes no extreme
                    hi = max(hi, vm[u] >> 16);
                }
            }
        tA[t] = sum;
        __shared__ int32_t tMm[kNT];
        tMm[t] = lo | (hi << 16);
        __syncthreads();
        if (t < CS) {
            for (int g2 = 1; g2 < ng; g2++) {
                const int i = g2 * CS + t;
                sum += tA[i];
                lo = min(lo, tMm[i] & 0xffff);
                hi = max(hi, tMm[i] >> 16);
            }
            // mu/2 = S1 2^(s_x - 1) / M, code floor(mu/2 2^(k_mu-1) + 1/2)
            sNmu[t] = (int32_t)clamp_k128(rhu128((i128)sum, s_x - 1 + (cf.k_mu - 1), (i128)st.M), cf.k_mu);
            sSum[t] = sum;
            sLo[t] = lo - 128;
            sHi[t] = hi - 128;
        }
    }
    __syncthreads();
    // Sum |D| over the channel's elements, D = q 2^(s_x - g) - n_mu 2^(e_mu - g)
    // (g = min(s_x, e_mu)), from int32 sums: with T the largest code whose D is
    // not positive, sum |D| = 2^(s_x - g) (2 S_gt - S) + n_mu 2^(e_mu - g) (M - 2 N_gt),
    // S_gt and N_gt the sum and count of the codes above T (the tail forms it)
    const int e_mu = 2 - cf.k_mu;
    const int gg = s_x < e_mu ? s_x : e_mu;
    int g, rsub;
    const bool active = stream_lane(st, g, rsub);
    int32_t sg[CPL], ng[CPL];
#pragma unroll
    for (int i = 0; i < CPL; i++) { sg[i] = 0; ng[i] = 0; }
    if (active) {
        int c0 = blockIdx.y * st.CS + g * CPL;
        int32_t T[CPL];
#pragma unroll
        for (int i = 0; i < CPL; i++) {
            const int64_t off = (int64_t)sNmu[g * CPL + i] * ((int64_t)1 << (e_mu - gg));
            const int64_t t = off >> (s_x - gg);          // floor(off / 2^(s_x - g))
            T[i] = (int32_t)(t < -129 ? -129 : (t > 127 ? 127 : t));
        }
        stream_rows<CPL, 4>(st, x, c0, rsub, [&](int64_t, const Vec<CPL>& v) {
#pragma unroll
            for (int i = 0; i < CPL; i++) {
                const int q = sbyte(v.w[i >> 2], i & 3);
                const bool up = q > T[i];
                sg[i] += up ? q : 0;
                ng[i] += up ? 1 : 0;
            }
        });
    }
    with_g(st.G, [&](auto gc) {
        constexpr int GG = decltype(gc)::value;
#pragma unroll
        for (int i = 0; i < CPL; i++) {
            sg[i] = fold_g<GG>(sg[i], OpAdd());
            ng[i] = fold_g<GG>(ng[i], OpAdd());
        }
    });
    if (fold) {
        const int wv = threadIdx.x >> 6;
        if ((int)(threadIdx.x & 63) < st.G) {
#pragma unroll
            for (int i = 0; i < CPL; i++) {
                wst[wv * 128 + g * CPL + i] = sg[i];
                wst[(kWaves + wv) * 128 + g * CPL + i] = ng[i];
            }
        }
        __syncthreads();
        if ((int)threadIdx.x < st.CS) {
            int32_t bs = 0, bn = 0;
#pragma unroll 4
            for (int v = 0; v < kWaves; v++) {
                bs += wst[v * 128 + threadIdx.x];
                bn += wst[(kWaves + v) * 128 + threadIdx.x];
            }
            sSg[threadIdx.x] = bs;
            sNg[threadIdx.x] = bn;
        }
    } else if (active && group_leader(st.G)) {
#pragma unroll
        for (int i = 0; i < CPL; i++) {
            atomicAdd(&sSg[g * CPL + i], sg[i]);
            atomicAdd(&sNg[g * CPL + i], ng[i]);
        }
    }
    __syncthreads();
    // one 8-byte partial per channel: the sum (low half) and the count (high half)
    if ((int)threadIdx.x < st.CS)
        st_x(&w.p_abs[(int64_t)blockIdx.x * st.C + blockIdx.y * st.CS + threadIdx.x],
             (long long)(((uint64_t)(uint32_t)sNg[threadIdx.x] << 32) | (uint32_t)sSg[threadIdx.x]));
    if (!arrive_last(w.ctr + 1 + blockIdx.y, gridDim.x)) return;
    // slice tail: sigma (Eq. 13-14), the denominator and this channel's bound on max|xhat|
    const int CS = st.CS, ngr = kNT / CS, t = threadIdx.x, ch = t % CS, grp = t / CS;
    const int64_t cb = (int64_t)blockIdx.y * CS;
    const int e_sig = 2 - cf.k_sigma;
    {
        long long acc_s = 0, acc_n = 0;
        if (grp < ngr)
            for (int b0 = grp; b0 < st.gx; b0 += kTailU * ngr) {
                long long va[kTailU];
#pragma unroll
                for (int u = 0; u < kTailU; u++) {
                    const int b = b0 + u * ngr;
                    va[u] = ld_x(&w.p_abs[(int64_t)(b < st.gx ? b : b0) * st.C + cb + ch]);
                }
#pragma unroll
                for (int u = 0; u < kTailU; u++)
                    if (b0 + u * ngr < st.gx) {
                        acc_s += (int32_t)(uint32_t)((uint64_t)va[u] & 0xffffffffu);
                        acc_n += (int32_t)(uint32_t)((uint64_t)va[u] >> 32);
                    }
            }
        tA[t] = acc_s;
        __syncthreads();
        if (t < CS)
            for (int g2 = 1; g2 < ngr; g2++) acc_s += tA[g2 * CS + t];
        __syncthreads();
        tA[t] = acc_n;
        __syncthreads();
        if (t < CS) {
            for (int g2 = 1; g2 < ngr; g2++) acc_n += tA[g2 * CS + t];
            const int64_t c = cb + t;
            const i128 mulq = pow2_128(s_x - gg), off = (i128)sNmu[t] * pow2_128(e_mu - gg);
            const i128 acc = mulq * (2 * (i128)acc_s - (i128)sSum[t]) + off * ((i128)st.M - 2 * (i128)acc_n);
            // sigma/2 = sumabs 2^(g-1) / M ; n_sigma = floor(sigma/2 2^(k_sigma-1) + 1/2)
            int32_t ns = (int32_t)clamp_k128(rhu128(acc, gg - 1 + (cf.k_sigma - 1), (i128)st.M), cf.k_sigma);
            int32_t den = ns + cf.eps_code;
            if (den < 1) den = 1;
            sv.n_sigma[c] = ns;
            sv.den[c] = den;
            const int32_t nm = sNmu[t];
            sv.n_mu[c] = nm;
            sv.qmin[c] = sLo[t];
            sv.qmax[c] = sHi[t];
            int best = kSentinelLo;
            const int qs[2] = {sLo[t], sHi[t]};
            for (int k = 0; k < 2; k++) {          // xhat is linear in q: extremes at qmin / qmax
                const int64_t D = bn_D(qs[k], s_x, nm, e_mu);
                if (D == 0) continue;
                const int e = ceil_pow2_exp128(abs128((i128)D), (i128)den) + gg - e_sig;
                best = e > best ? e : best;
            }
            tA[t] = best;                          // slot t is read by thread t only above
        }
    }
    __syncthreads();
    int bmax = kSentinelLo;
    for (int i = t; i < CS; i += kNT) bmax = max(bmax, (int)tA[i]);
    bmax = block_max_nt(bmax, rb);
    if (t == 0) w.sbmax[blockIdx.y] = bmax;
}

// max of n per-slice values, by every thread of the block (kSentinelLo if n = 0)
__device__ __forceinline__ int32_t slices_max(const int32_t* a, int n, int32_t* sh)
{
    int32_t m = kSentinelLo;
    for (int i = threadIdx.x; i < n; i += blockDim.x) m = max(m, a[i]);
    for (int o = 32; o > 0; o >>= 1) m = max(m, __shfl_xor(m, o, 64));
    __syncthreads();
    if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = m;
    __syncthreads();
    m = sh[0];
    for (int k = 1; k < (int)(blockDim.x >> 6); k++) m = max(m, sh[k]);
    return m;
}

// shift of a channel's staged A values: max(0, r_c - 1), r_c = bitlen(max) -
// (k_A - 1) the Q_A shift of the channel's own max |ReLU(y)|
__device__ __forceinline__ int ystg_shift(uint64_t maxy, int kA)
{
    const int rc = maxy ? bitlen_u64(maxy) - (kA - 1) : 0;
    return rc > 1 ? rc - 1 : 0;
}

// per (channel, code): xhat code, y, flags and the backward's entry; per
// channel: the sgn and ReLU thresholds and max |ReLU(y)| over the occupied
// codes (y is monotone in q, so over qmin and qmax)
__global__ __launch_bounds__(256) void k_bnf_fin2(const int32_t* x_exp, int nslices, FwdWs w, Saved sv, BnCfg cf,
                                                  const int8_t* gamma_q, const int8_t* beta_q)
{
    __shared__ int32_t rsh[4];
    const int c = blockIdx.x;
    const int q = (int)threadIdx.x - 128;
    int32_t s_x = *x_exp;
    if (!sx_ok(s_x)) return;
    int b = slices_max(w.sbmax, nslices, rsh);
    if (b == kSentinelLo) b = 0;
    if (c == 0 && threadIdx.x == 0) *w.b_glob = b;
    const FwdExps e = fwd_exps(s_x, b, cf);
    const int64_t D = bn_D(q, s_x, sv.n_mu[c], e.e_mu);
    const i128 nx = fwd_xcode(D, sv.den[c], b, e);
    const i128 Y = fwd_y(nx, gamma_q[c], beta_q[c], e);
    const int idx = c * 256 + threadIdx.x;
    sv.xcode[idx] = (int16_t)nx;
    const int sg = (D > 0) - (D < 0);
    sv.flags[idx] = (uint8_t)((Y > 0 ? 1 : 0) | ((sg + 1) << 1));
    sv.btab[c * 256 + (q & 255)] = ((uint32_t)(uint16_t)(int16_t)nx << 16) | ((uint32_t)(sg & 3) << 8) |
                                   ((uint32_t)(sg != 0) << 10) | (Y > 0 ? 1u : 0u);
    // thresholds (least code with D >= 0, least with D > 0, code range with y > 0)
    // and the channel's max |ReLU(y)| over its occupied code extremes, by block
    // reductions: same-address atomics would serialize 256 updates per channel
    int v0 = D >= 0 ? q : 128, v1 = D > 0 ? q : 128, v2 = Y > 0 ? q : 128, v3 = Y > 0 ? q : -129;
    const i128 Yr = cf.relu && Y < 0 ? 0 : Y;
    uint64_t ay = (q == sv.qmin[c] || q == sv.qmax[c]) ? (uint64_t)abs128(Yr) : 0;
    for (int o = 32; o > 0; o >>= 1) {
        v0 = min(v0, __shfl_xor(v0, o)); v1 = min(v1, __shfl_xor(v1, o));
        v2 = min(v2, __shfl_xor(v2, o)); v3 = max(v3, __shfl_xor(v3, o));
        const uint64_t t = __shfl_xor(ay, o);
        ay = t > ay ? t : ay;
    }
    __shared__ int32_t red[4][4];
    __shared__ uint64_t ry[4];
    const int wv = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) { red[wv][0] = v0; red[wv][1] = v1; red[wv][2] = v2; red[wv][3] = v3; ry[wv] = ay; }
    __syncthreads();
    __shared__ uint64_t s_ay;
    if (threadIdx.x == 0) {
        for (int k = 1; k < 4; k++) {
            v0 = min(v0, red[k][0]); v1 = min(v1, red[k][1]); v2 = min(v2, red[k][2]); v3 = max(v3, red[k][3]);
            ay = ry[k] > ay ? ry[k] : ay;
        }
        sv.t0[c] = v0; sv.p0[c] = v1; sv.mlo[c] = v2; sv.mhi[c] = v3;
        w.maxYc[c] = ay;
        s_ay = ay;
    }
    __syncthreads();
    // ReLU(y) floored by 2^t_c, t_c = max(0, r_c - 1) with r_c the Q_A shift
    // this channel's own maximum would give: below 2^k_A in magnitude for the
    // occupied codes (clamped elsewhere, where the output pass never looks)
    const int tc = ystg_shift(s_ay, cf.k_A);
    i128 z = tc ? (Yr >> tc) : Yr;
    z = z > 32767 ? 32767 : (z < -32767 ? -32767 : z);
    sv.ystg[idx] = (int16_t)z;
}

// Output pass.  Every block first takes Q_A's shift r from the channels'
// maxima (block (0, 0) writes the output exponent and the saved header), then
//   * writes its share of the saved A codes, exactly from the xhat codes (the
//     table the inference path applies, every code included);
//   * builds its channels' gather table from the staged values:
//     code = ((z >> (r - 1 - t_c)) + 1) >> 1, the half-up rounding of
//     ReLU(y) by 2^r (half-up rounding of floor(v / 2^t) by 2^(r - t) equals
//     that of v for t < r), two codes per packed 16-bit operation.
template <int CPL>
__global__ __launch_bounds__(1024) void k_bnf_apply(const int8_t* __restrict__ x, int8_t* __restrict__ y,
                                                   Stream st, Saved sv, FwdWs w, BnCfg cf, const int32_t* x_exp,
                                                   const int8_t* gamma_q, const int8_t* beta_q, int32_t* y_exp)
{
    __shared__ __attribute__((aligned(16))) int8_t lut[128 * kRowB];
    __shared__ uint64_t rmax[kNT / 64];
    uint64_t M = 0;
    for (int k = threadIdx.x; k < st.C; k += kNT) M = w.maxYc[k] > M ? w.maxYc[k] : M;
    for (int o = 32; o > 0; o >>= 1) {
        const uint64_t t = __shfl_xor(M, o);
        M = t > M ? t : M;
    }
    if ((threadIdx.x & 63) == 0) rmax[threadIdx.x >> 6] = M;
    __syncthreads();
    M = rmax[0];
    for (int k = 1; k < kNT / 64; k++) M = rmax[k] > M ? rmax[k] : M;
    const int r = M ? bitlen_u64(M) - (cf.k_A - 1) : 0;
    int32_t s_x = *x_exp;
    const bool ok = sx_ok(s_x);
    if (!ok) s_x = -14;          // outputs unspecified; keeps the shifts defined
    const int b = *w.b_glob;
    const FwdExps e = fwd_exps(s_x, b, cf);
    if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0 && ok) {
        *y_exp = e.e_y + r;
        sv.hdr[0] = b;
        sv.hdr[1] = e.e_y;
        sv.hdr[2] = e.e_y + r;
        sv.hdr[3] = s_x;
    }
    if (ok) {
        const int64_t nall = (int64_t)st.C * 256, nb = (int64_t)gridDim.x * gridDim.y;
        const int64_t per = (nall + nb - 1) / nb;
        const int64_t i0 = ((int64_t)blockIdx.y * gridDim.x + blockIdx.x) * per;
        for (int64_t i = i0 + threadIdx.x; i < i0 + per && i < nall; i += kNT) {
            const int c = (int)(i >> 8);
            i128 Yv = fwd_y((i128)sv.xcode[i], gamma_q[c], beta_q[c], e);
            if (cf.relu && Yv < 0) Yv = 0;
            sv.acode[i] = (int8_t)sq_code((long long)Yv, r, cf.k_A);
        }
    }
    if (!ok) {
        for (int i = threadIdx.x; i < st.CS * kRowB; i += kNT) lut[i] = 0;
    } else {
        const short lim = (short)((1 << (cf.k_A - 1)) - 1);
        const int16_t* src = sv.ystg + (int64_t)blockIdx.y * st.CS * 256;
        for (int v = threadIdx.x; v < st.CS * 32; v += kNT) {       // eight codes per step
            const int i0 = v * 8, row = i0 >> 8, col = i0 & 255;
            const int tc = ystg_shift(w.maxYc[blockIdx.y * st.CS + row], cf.k_A);
            const int4 q = *(const int4*)(src + i0);
            const int qw[4] = {q.x, q.y, q.z, q.w};
            uint32_t ow[2] = {0, 0};
            const short sh = (short)(r > 0 ? min(r - 1 - tc, 15) : 0), up = (short)(r < 0 ? -r : 0);
#pragma unroll
            for (int h = 0; h < 4; h++) {
                short2v zv = __builtin_bit_cast(short2v, qw[h]);
                if (r > 0) zv = ((zv >> sh) + (short)1) >> (short)1;
                else zv = zv << up;
                zv = zv > lim ? lim : zv;
                zv = zv < (short)-lim ? (short)-lim : zv;
                const uint32_t bb = ((uint32_t)(uint16_t)zv.x & 0xffu) | (((uint32_t)(uint16_t)zv.y & 0xffu) << 8);
                ow[h >> 1] |= bb << (16 * (h & 1));
            }
            *(uint32_t*)(lut + row * kRowB + col) = ow[0];
            *(uint32_t*)(lut + row * kRowB + col + 4) = ow[1];
        }
    }
    __syncthreads();
    int g, rsub;
    if (!stream_lane(st, g, rsub)) return;
    const int c0 = blockIdx.y * st.CS + g * CPL;
    const int8_t* l = lut + g * CPL * kRowB + 128;
    stream_rows<CPL, 4>(st, x, c0, rsub, [&](int64_t r, const Vec<CPL>& v) {
        Vec<CPL> o;
#pragma unroll
        for (int j = 0; j < CPL / 4; j++) {
            uint32_t ow = 0;
#pragma unroll
            for (int i = 0; i < 4; i++)
                ow |= (uint32_t)(uint8_t)l[(j * 4 + i) * kRowB + sbyte(v.w[j], i)] << (8 * i);
            o.w[j] = ow;
        }
        vstore<CPL>(y + r * st.C + c0, o);
    });
}

// ---------------------------------------------------------------------------
// backward workspace
// ---------------------------------------------------------------------------
struct BwdWs {
    uint32_t* ctr;                   // arrival counters
    int32_t* smax;                   // [slices] bound on E1's exponent over each slice's channels
    int32_t* smaxF;                  // [slices] max |gamma delta| over each slice's channels (rounding E2)
    int32_t *p_sd, *p_z, *p_mmA, *p_mmB;   // [gx][C] partials (per-class extremes packed as bytes)
    long long *p_sdn, *p_sf, *p_sfn; // [gx][C]
    long long *sd, *sdn, *sf, *sfn;  // [C] reduced
    int32_t *Z, *mm;                 // [C], [C][6]
    int8_t* lut;                     // [C][3][256] dx codes (rounding E2)
    int32_t* cbnd;                   // [C] each channel's bound on E1's exponent (exact E2)
    int16_t* lutq;                   // [C][3][256] dx values at the channel's own bound (exact E2)
};

size_t bwd_ws_bytes(const Stream& st)
{
    size_t pc = (size_t)st.gx * st.C, C = (size_t)st.C;
    return ctr_bytes(st.C) + 2 * align256(C) + 4 * align256(pc * 4) + 3 * align256(pc * 8) +
           4 * align256(C * 8) + align256(C * 4) + align256(C * 24) + align256(C * 768) + align256(C * 4) +
           align256(C * 768 * 2);
}

BwdWs bwd_ws_map(void* base, const Stream& st)
{
    char* p = (char*)base;
    size_t pc = (size_t)st.gx * st.C, C = (size_t)st.C;
    BwdWs w;
    w.ctr = (uint32_t*)p; p += ctr_bytes(st.C);
    w.smax = (int32_t*)p; p += align256(C);          // slices <= C / 4
    w.smaxF = (int32_t*)p; p += align256(C);
    w.p_sd = (int32_t*)p; p += align256(pc * 4);
    w.p_z = (int32_t*)p; p += align256(pc * 4);
    w.p_mmA = (int32_t*)p; p += align256(pc * 4);
    w.p_mmB = (int32_t*)p; p += align256(pc * 4);
    w.p_sdn = (long long*)p; p += align256(pc * 8);
    w.p_sf = (long long*)p; p += align256(pc * 8);
    w.p_sfn = (long long*)p; p += align256(pc * 8);
    w.sd = (long long*)p; p += align256(C * 8);
    w.sdn = (long long*)p; p += align256(C * 8);
    w.sf = (long long*)p; p += align256(C * 8);
    w.sfn = (long long*)p; p += align256(C * 8);
    w.Z = (int32_t*)p; p += align256(C * 4);
    w.mm = (int32_t*)p; p += align256(C * 24);
    w.lut = (int8_t*)p; p += align256(C * 768);
    w.cbnd = (int32_t*)p; p += align256(C * 4);
    w.lutq = (int16_t*)p;
    return w;
}

// sgn class (sgn + 1) and ReLU mask of an input code from the thresholds
struct Thr {
    int t0, p0, mlo, mhi;
};

__device__ __forceinline__ int thr_cls(const Thr& t, int q) { return 1 + (q >= t.p0) - (q < t.t0); }
__device__ __forceinline__ bool thr_mask(const Thr& t, int q) { return q >= t.mlo && q <= t.mhi; }

// Copy the channel slice's per-(channel, code) entries (saved by the forward)
// into LDS rows of kRowW dwords, all loads of a thread issued before the first
// store.  The ReLU bit becomes a mask byte in bits 0..7 (0xff passes delta).
// With `lut_off` the upper half is replaced by the offset of the entry's
// sgn-class row in the slice's dx-code tables (three rows of kRowB bytes per
// channel, +128 for the signed delta).
constexpr int kTabV = 64 * 256 / 4 / kNT;    // 16-byte pieces per thread (CS <= 64)
__device__ __forceinline__ void load_bwd_tab(uint32_t* tab, const uint32_t* src, int CS, int relu,
                                             bool lut_off)
{
    const int nv = CS * 64;
    uint4 v[kTabV];
#pragma unroll
    for (int k = 0; k < kTabV; k++) {
        const int i = threadIdx.x + k * kNT;
        if (i < nv) v[k] = ((const uint4*)src)[i];
    }
#pragma unroll
    for (int k = 0; k < kTabV; k++) {
        const int i = threadIdx.x + k * kNT;
        if (i < nv) {
            uint32_t e[4] = {v[k].x, v[k].y, v[k].z, v[k].w};
#pragma unroll
            for (int j = 0; j < 4; j++) {
                const uint32_t m = (!relu || (e[j] & 1)) ? 0xffu : 0u;
                if (lut_off) {
                    const int cl = (4 * i + j) >> 8;
                    const int sg = ((int)(e[j] << 22)) >> 30;
                    e[j] = ((uint32_t)((cl * 3 + sg + 1) * kRowB + 128) << 16) | m;
                } else {
                    e[j] = (e[j] & 0xffffff00u) | m;
                }
            }
            uint32_t* d = tab + (i >> 6) * kRowW + (i & 63) * 4;
            d[0] = e[0]; d[1] = e[1]; d[2] = e[2]; d[3] = e[3];
        }
    }
}

// Per-class extremes of the masked delta travel between blocks as bytes:
// low ends as lo + 128 (255 for an empty class), high ends as hi + 128 (0 for
// an empty class), so a byte-wise min / max merges them and an empty class
// still reads lo > hi.  A = (lo, hi) of classes -1 and 0, B = (lo, hi) of +1.
__device__ __forceinline__ uint32_t pk_lo(int v) { return v > 127 ? 255u : (uint32_t)(v + 128); }
__device__ __forceinline__ uint32_t pk_hi(int v) { return v < -128 ? 0u : (uint32_t)(v + 128); }
__device__ __forceinline__ void mm_pack(const int* mm, uint32_t& A, uint32_t& B)
{
    A = pk_lo(mm[0]) | pk_hi(mm[1]) << 8 | pk_lo(mm[2]) << 16 | pk_hi(mm[3]) << 24;
    B = pk_lo(mm[4]) | pk_hi(mm[5]) << 8;
}
__device__ __forceinline__ void mm_merge(uint32_t A, uint32_t B, int* lo3, int* hi3)
{
    lo3[0] = min(lo3[0], (int)(A & 0xff)); hi3[0] = max(hi3[0], (int)((A >> 8) & 0xff));
    lo3[1] = min(lo3[1], (int)((A >> 16) & 0xff)); hi3[1] = max(hi3[1], (int)(A >> 24));
    lo3[2] = min(lo3[2], (int)(B & 0xff)); hi3[2] = max(hi3[2], (int)((B >> 8) & 0xff));
}

// Pass 1: sum delta, sum delta*xhat, sum sgn and the per-sgn-class extremes of
// the masked delta d.  The extremes come from four keys per element, d +- 1024 s
// and d +- 1024 |s| (s = sgn in {-1, 0, 1}, |d| <= 128): the minimum of d + 1024 s
// lies in class -1 whenever that class is present, its maximum in class +1, and
// likewise for the others, so six min/max updates replace per-class selects.
constexpr int kKey = 1024;
constexpr int kKeyInit = 4 * kKey;
struct BnbOut {
    const int32_t* dy_exp;
    const int8_t* gamma_q;
    int64_t *dgamma, *dbeta;
    int32_t *dgamma_exp, *dbeta_exp, *dx_exp, *dev_status;
};

__device__ __forceinline__ void bnb_round_tail1(uint32_t* lds, const Stream& st, const BwdWs& w, const Saved& sv,
                                                const BnCfg& cf, const BnbOut& o);

// Block totals per channel.  When the G lanes of a row (G = CS / 4) are a
// power of two, the lanes of a wave that hold the same channels are folded
// with shuffles and the 16 wave totals of each channel are staged in LDS
// (the caller's table space, no longer read) and summed by one thread per
// channel: LDS atomics from every wave onto the same channel slots serialize
// and cost several microseconds per block.  Other widths use LDS atomics.

template <int TAIL>                      // 1: exact E2, 2: rounding E2
__global__ __launch_bounds__(1024) void k_bnb_stats(const int8_t* __restrict__ dy,
                                                   const int8_t* __restrict__ x, Stream st, BwdWs w,
                                                   Saved sv, BnCfg cf, BnbOut out)
{
    const int relu = cf.relu;
    __shared__ __attribute__((aligned(16))) uint32_t tab[64 * kRowW];
    __shared__ unsigned long long sSdn[64];
    __shared__ int32_t sSd[64], sZ[64], sMM[64 * 6];
    const int64_t cbase = (int64_t)blockIdx.y * st.CS;
    const bool fold = (st.G & (st.G - 1)) == 0 && st.G <= 64;
    load_bwd_tab(tab, sv.btab + cbase * 256, st.CS, relu, false);
    if (!fold && (int)threadIdx.x < st.CS) {
        sSdn[threadIdx.x] = 0; sSd[threadIdx.x] = 0; sZ[threadIdx.x] = 0;
        for (int k = 0; k < 3; k++) { sMM[threadIdx.x * 6 + 2 * k] = 1000; sMM[threadIdx.x * 6 + 2 * k + 1] = -1000; }
    }
    __syncthreads();
    int g, rsub;
    const bool active = stream_lane(st, g, rsub);
    int32_t sd[4] = {0, 0, 0, 0}, z[4] = {0, 0, 0, 0};
    int64_t sdn[4] = {0, 0, 0, 0};
    // key extremes: min(d + 1024 s), max(d + 1024 s), min(d - 1024 s), max(d - 1024 s),
    // min(d + 1024 |s|), max(d - 1024 |s|)
    int32_t kmn0[4], kmx0[4], kmn1[4], kmx1[4], kmn2[4], kmx3[4];
#pragma unroll
    for (int i = 0; i < 4; i++) {
        kmn0[i] = kmn1[i] = kmn2[i] = kKeyInit;
        kmx0[i] = kmx1[i] = kmx3[i] = -kKeyInit;
    }
    if (active) {
        const int c0 = (int)cbase + g * 4;
        const uint32_t* tb = tab + g * 4 * kRowW;
        const int64_t step = (int64_t)gridDim.x * st.rpi;
        auto elem = [&](uint32_t wx, uint32_t wd, int32_t* sdn32) {
#pragma unroll
            for (int i = 0; i < 4; i++) {
                const uint32_t e = tb[i * kRowW + ((wx >> (8 * i)) & 0xff)];
                const int dm = sbyte(wd, i) & (int)(int8_t)(e & 0xff);
                const int sg = ((int)(e << 22)) >> 30;            // bits 8..9, signed
                const int ab = (int)((e >> 10) & 1);
                sd[i] += dm;
                sdn32[i] += dm * ((int)e >> 16);
                z[i] += sg;
                const int k0 = dm + sg * kKey, k1 = dm - sg * kKey;
                const int k2 = dm + ab * kKey, k3 = dm - ab * kKey;
                kmn0[i] = min(kmn0[i], k0); kmx0[i] = max(kmx0[i], k0);
                kmn1[i] = min(kmn1[i], k1); kmx1[i] = max(kmx1[i], k1);
                kmn2[i] = min(kmn2[i], k2); kmx3[i] = max(kmx3[i], k3);
            }
        };
        // full groups of U rows (all in range), next group's loads issued
        // before this group's arithmetic; then the remaining rows one by one
        constexpr int U = 4;
        int64_t r = (int64_t)blockIdx.x * st.rpi + rsub;
        const int64_t full_end = st.M - (U - 1) * step;
        uint32_t vx[U], vd[U], nx[U], nd[U];
        auto load = [&](int64_t r0, uint32_t* ax, uint32_t* ad) {
#pragma unroll
            for (int u = 0; u < U; u++) {
                ax[u] = *(const uint32_t*)(x + (r0 + u * step) * st.C + c0);
                ad[u] = *(const uint32_t*)(dy + (r0 + u * step) * st.C + c0);
            }
        };
        if (r < full_end) load(r, vx, vd);
        while (r < full_end) {
            const int64_t rn = r + U * step;
            if (rn < full_end) load(rn, nx, nd);
            int32_t sdn32[4] = {0, 0, 0, 0};
#pragma unroll
            for (int u = 0; u < U; u++) elem(vx[u], vd[u], sdn32);
#pragma unroll
            for (int i = 0; i < 4; i++) sdn[i] += sdn32[i];
#pragma unroll
            for (int u = 0; u < U; u++) { vx[u] = nx[u]; vd[u] = nd[u]; }
            r = rn;
        }
        for (; r < st.M; r += step) {
            int32_t sdn32[4] = {0, 0, 0, 0};
            elem(*(const uint32_t*)(x + r * st.C + c0), *(const uint32_t*)(dy + r * st.C + c0), sdn32);
#pragma unroll
            for (int i = 0; i < 4; i++) sdn[i] += sdn32[i];
        }
    }
    // decode the keys into (min, max) per class; an empty class gives (1000, -1000)
    int32_t mm[4][6];
#pragma unroll
    for (int i = 0; i < 4; i++) {
        mm[i][0] = kmn0[i] <= -kKey + 128 ? kmn0[i] + kKey : 1000;     // class -1
        mm[i][1] = kmx1[i] >= kKey - 128 ? kmx1[i] - kKey : -1000;
        mm[i][2] = kmn2[i] <= 128 ? kmn2[i] : 1000;                     // class 0
        mm[i][3] = kmx3[i] >= -128 ? kmx3[i] : -1000;
        mm[i][4] = kmn1[i] <= -kKey + 128 ? kmn1[i] + kKey : 1000;     // class +1
        mm[i][5] = kmx0[i] >= kKey - 128 ? kmx0[i] - kKey : -1000;
    }
    with_g(st.G, [&](auto gc) {
        constexpr int GG = decltype(gc)::value;
#pragma unroll
        for (int i = 0; i < 4; i++) {
            sd[i] = fold_g<GG>(sd[i], OpAdd());
            sdn[i] = fold_g<GG>(sdn[i], OpAdd());
            z[i] = fold_g<GG>(z[i], OpAdd());
#pragma unroll
            for (int k = 0; k < 3; k++) {
                mm[i][2 * k] = fold_g<GG>(mm[i][2 * k], OpMin());
                mm[i][2 * k + 1] = fold_g<GG>(mm[i][2 * k + 1], OpMax());
            }
        }
    });
    const int t = threadIdx.x;
    int32_t bsd = 0, bz = 0;
    long long bsdn = 0;
    int bmm[6] = {1000, -1000, 1000, -1000, 1000, -1000};
    if (fold) {
        __syncthreads();                                  // every wave is done with the table
        int32_t* wsd = (int32_t*)tab;                     // [kWaves][64] each
        int32_t* wz = wsd + kWaves * 64;
        int32_t* wmm = wz + kWaves * 64;                  // [6][kWaves][64]
        long long* wsdn = (long long*)(wmm + 6 * kWaves * 64);
        const int wv = t >> 6;
        if ((t & 63) < st.G) {
#pragma unroll
            for (int i = 0; i < 4; i++) {
                const int s = wv * 64 + g * 4 + i;
                wsd[s] = sd[i]; wz[s] = z[i]; wsdn[s] = sdn[i];
#pragma unroll
                for (int k = 0; k < 6; k++) wmm[k * kWaves * 64 + s] = mm[i][k];
            }
        }
        __syncthreads();
        if (t < st.CS) {
#pragma unroll 4
            for (int v = 0; v < kWaves; v++) {
                const int s = v * 64 + t;
                bsd += wsd[s]; bz += wz[s]; bsdn += wsdn[s];
#pragma unroll
                for (int k = 0; k < 6; k++) {
                    const int m = wmm[k * kWaves * 64 + s];
                    bmm[k] = (k & 1) ? max(bmm[k], m) : min(bmm[k], m);
                }
            }
        }
    } else {
        if (active && group_leader(st.G)) {
#pragma unroll
            for (int i = 0; i < 4; i++) {
                int cl = g * 4 + i;
                atomicAdd(&sSd[cl], sd[i]);
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
        if (t < st.CS) {
            bsd = sSd[t]; bz = sZ[t]; bsdn = (long long)sSdn[t];
            for (int k = 0; k < 6; k++) bmm[k] = sMM[t * 6 + k];
        }
    }
    if (t < st.CS) {
        uint32_t A, B;
        mm_pack(bmm, A, B);
        if constexpr (TAIL == 1) {
            // [slice][block][channel of the slice]: one contiguous row per block
            const int64_t o = ((int64_t)blockIdx.y * st.gx + blockIdx.x) * st.CS + t;
            w.p_sd[o] = bsd;
            w.p_sdn[o] = bsdn;
            w.p_z[o] = bz;
            w.p_mmA[o] = (int32_t)A;
            w.p_mmB[o] = (int32_t)B;
        } else {
            const int64_t o = (int64_t)blockIdx.x * st.C + cbase + t;
            st_x(&w.p_sd[o], bsd);
            st_x(&w.p_sdn[o], bsdn);
            st_x(&w.p_z[o], bz);
            st_x(&w.p_mmA[o], (int32_t)A);
            st_x(&w.p_mmB[o], (int32_t)B);
        }
    }
    if constexpr (TAIL == 2) {
        if (arrive_last(w.ctr + 1 + blockIdx.y, gridDim.x)) {
            __syncthreads();                              // the staging above may still be read
            bnb_round_tail1(tab, st, w, sv, cf, out);
        }
    }
}


// E2's requant shift from max |gamma delta| (the slices' maxima)
__device__ __forceinline__ int bnb_r2_of(int32_t maxF, const BnCfg& cf)
{
    return maxF > 0 ? bitlen_u64((uint64_t)maxF) - (cf.k_E2 - 1) : 0;
}

__device__ __forceinline__ void bnb_round_tail2(uint32_t* lds, const Stream& st, const BwdWs& w,
                                                const Saved& sv, const BnCfg& cf, const BnbOut& o, int r2);

// pass 2 (only when E2's quantizer rounds): sum f and f*n_xhat; the tails
// reduce them and give each slice's bound on E1's exponent
__global__ __launch_bounds__(1024) void k_bnb_stats2(const int8_t* __restrict__ dy,
                                                    const int8_t* __restrict__ x, Stream st, BwdWs w,
                                                    Saved sv, BnCfg cf, BnbOut out)
{
    const int8_t* gamma_q = out.gamma_q;
    __shared__ __attribute__((aligned(16))) int16_t xc[64 * 256];
    __shared__ int16_t ft[64 * 256];                  // f = SQ(gamma_q d, k_E2) per (channel, d)
    __shared__ Thr thr[64];
    __shared__ unsigned long long sF[64], sFn[64];
    __shared__ int32_t rsh[kNT / 64];
    const int64_t cbase = (int64_t)blockIdx.y * st.CS;
    {
        copy_to_lds<64 * 512 / 16 / kNT>((uint4*)xc, (const uint4*)(sv.xcode + cbase * 256), st.CS * 32);
    }
    if ((int)threadIdx.x < st.CS) {
        int c = (int)cbase + threadIdx.x;
        thr[threadIdx.x] = Thr{sv.t0[c], sv.p0[c], cf.relu ? sv.mlo[c] : -1000, cf.relu ? sv.mhi[c] : 1000};
        sF[threadIdx.x] = 0; sFn[threadIdx.x] = 0;
    }
    // |f| < 2^(k_E2-1) <= 2^13 on this path
    const int r2 = bnb_r2_of(slices_max(w.smaxF, (int)gridDim.y, rsh), cf);
    for (int e = threadIdx.x; e < st.CS * 256; e += blockDim.x)
        ft[e] = (int16_t)sq_code((int64_t)gamma_q[cbase + (e >> 8)] * ((e & 255) - 128), r2, cf.k_E2);
    __syncthreads();
    int g, rsub;
    const bool active = stream_lane(st, g, rsub);
    int64_t sf[4] = {0, 0, 0, 0}, sfn[4] = {0, 0, 0, 0};
    if (active) {
        const int c0 = (int)cbase + g * 4;
        Thr t[4];
#pragma unroll
        for (int i = 0; i < 4; i++) t[i] = thr[g * 4 + i];
        stream_rows2<4, 8>(st, x, dy, c0, rsub, [&](int64_t, const Vec<4>& vxx, const Vec<4>& vdd) {
            const uint32_t vx = vxx.w[0], vd = vdd.w[0];
#pragma unroll
            for (int i = 0; i < 4; i++) {
                int q = sbyte(vx, i);
                int d = thr_mask(t[i], q) ? sbyte(vd, i) : 0;
                const int f = ft[(g * 4 + i) * 256 + d + 128];
                sf[i] += f;
                sfn[i] += f * (int)xc[(g * 4 + i) * 256 + q + 128];     // |f x| < 2^28
            }
        });
    }
    with_g(st.G, [&](auto gc) {
        constexpr int GG = decltype(gc)::value;
#pragma unroll
        for (int i = 0; i < 4; i++) {
            sf[i] = fold_g<GG>(sf[i], OpAdd());
            sfn[i] = fold_g<GG>(sfn[i], OpAdd());
        }
    });
    if (active && group_leader(st.G)) {
#pragma unroll
        for (int i = 0; i < 4; i++) {
            atomicAdd(&sF[g * 4 + i], (unsigned long long)sf[i]);
            atomicAdd(&sFn[g * 4 + i], (unsigned long long)sfn[i]);
        }
    }
    __syncthreads();
    if ((int)threadIdx.x < st.CS) {
        int64_t o = (int64_t)blockIdx.x * st.C + cbase + threadIdx.x;
        st_x(&w.p_sf[o], (long long)sF[threadIdx.x]);
        st_x(&w.p_sfn[o], (long long)sFn[threadIdx.x]);
    }
    if (arrive_last(w.ctr + 1 + blockIdx.y, gridDim.x)) {
        __syncthreads();
        bnb_round_tail2((uint32_t*)xc, st, w, sv, cf, out, r2);
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

// exponents of a channel's bracket for E2's shift r2
__device__ __forceinline__ BnbChan bnb_chan_exps(int r2, int32_t dy_exp, const Saved& sv, const BnCfg& cf)
{
    BnbChan ch;
    ch.r2 = r2;
    ch.e_xh = sv.hdr[0] - (cf.k_xhat - 1);
    const int e_sig = 2 - cf.k_sigma, e_g = 2 - cf.k_gamma;
    const int s2 = dy_exp + e_g + r2;
    ch.Ebase = s2 - e_sig + (ch.e_xh < 0 ? ch.e_xh : 0);
    return ch;
}

__device__ __forceinline__ void bnb_exps_out(const Saved& sv, const BnCfg& cf, const BnbOut& o)
{
    const int32_t s_d = *o.dy_exp;
    if (s_d < -60 || s_d > 16) set_status(o.dev_status, ISEG_DEV_RANGE);
    *o.dbeta_exp = s_d;
    *o.dgamma_exp = s_d + sv.hdr[0] - (cf.k_xhat - 1);
}

// dx code table for every (sgn class, masked error code) of a channel
// (rounding E2): E1's exponent and E2's shift from the slices' maxima
__global__ __launch_bounds__(256) void k_bnb_lut(int64_t Mrows, int nslices, BwdWs w, Saved sv, BnCfg cf,
                                                 BnbOut o)
{
    __shared__ int32_t rsh[4];
    const int c = blockIdx.x;
    const int d = (int)threadIdx.x - 128;
    const int gq = o.gamma_q[c];
    const int r2 = bnb_r2_of(slices_max(w.smaxF, nslices, rsh), cf);
    int bdx = slices_max(w.smax, nslices, rsh);
    if (bdx == kSentinelLo) bdx = 0;
    if (c == 0 && threadIdx.x == 0) {
        *o.dx_exp = bdx - (cf.k_E1 - 1);
        bnb_exps_out(sv, cf, o);
    }
    BnbChan ch = bnb_chan_exps(r2, *o.dy_exp, sv, cf);
    ch.Sf = (i128)w.sf[c];
    ch.T = (i128)w.sfn[c];
    ch.Z = (i128)w.Z[c];
    const i128 M = Mrows;
    const i128 Dd = (i128)sv.den[c] * M * M;
    const int64_t f = d < -127 ? 0 : sq_code((int64_t)gq * d, ch.r2, cf.k_E2);
    for (int k = 0; k < 3; k++) {
        int8_t code = 0;
        if (d >= -127) {
            i128 B = bnb_bracket(f, k - 1, M, ch.Sf, ch.T, ch.Z, ch.e_xh);
            code = (int8_t)clamp_k128(rhu128(B, ch.Ebase + (cf.k_E1 - 1) - bdx, Dd), cf.k_E1);
        }
        w.lut[((int64_t)c * 3 + k) * 256 + threadIdx.x] = code;
    }
}

// ---------------------------------------------------------------------------
// Exact E2 (k_E2 >= 15, |gamma delta| <= 127^2 < 2^(k_E2-1)): E2's requant
// shift r2 is <= 0 and scales every term of the bracket and the exponent base
// by inverse powers of two, so dx, its exponent bound and its codes are those
// of r2 = 0, with f = gamma_q delta; the stats kernel's tails replace a
// separate per-channel pass.
// ---------------------------------------------------------------------------
// stats tail (exact E2).  Slice: the pass-1 sums, dgamma and dbeta of its
// channels and each channel's bound on max|dx| (|dx| is extreme at a class's
// extreme deltas: six candidates per channel, one thread each); the largest
// bound of the slice goes to smax for the table kernel, which takes E1's
// exponent as the largest over the slices.  `lds` is the stats table, no
// longer read once the block has arrived.
struct Tail1Lds {
    int32_t *sd, *z, *mm, *cand;        // [kNT], [kNT], [6][kNT], [6 * CS]
    long long* sdn;                     // [kNT]
    __device__ explicit Tail1Lds(uint32_t* lds)
    {
        sd = (int32_t*)lds; z = sd + kNT; mm = z + kNT;
        sdn = (long long*)(mm + 6 * kNT); cand = (int32_t*)(sdn + kNT);
    }
};

// the slice's pass-1 sums from all blocks' partials: w.sd / sdn / Z / mm,
// dgamma, dbeta, and the channel totals in the group-0 slots of the LDS table
__device__ __forceinline__ void bnb_tail_reduce1(uint32_t* lds, const Stream& st, const BwdWs& w,
                                                 const BnbOut& o)
{
    const int CS = st.CS, ng = kNT / CS, t = threadIdx.x, ch = t % CS, grp = t / CS;
    const Tail1Lds L(lds);
    int32_t* tSd = L.sd;
    int32_t* tZ = L.z;
    int32_t* tMM = L.mm;
    long long* tSdn = L.sdn;
    const int64_t cb = (int64_t)blockIdx.y * CS;
    int sd = 0, z = 0;
    long long sdn = 0;
    int lo3[3] = {255, 255, 255}, hi3[3] = {0, 0, 0};   // byte-coded extremes
    constexpr int U = 8;                    // partial rows whose loads are in flight together
    if (grp < ng)
        for (int b0 = grp; b0 < st.gx; b0 += U * ng) {
            int32_t vsd[U], vz[U], vA[U], vB[U];
            long long vsdn[U];
#pragma unroll
            for (int u = 0; u < U; u++) {
                const int b = b0 + u * ng;
                const int64_t q = (int64_t)(b < st.gx ? b : b0) * st.C + cb + ch;
                vsd[u] = ld_x(&w.p_sd[q]);
                vsdn[u] = ld_x(&w.p_sdn[q]);
                vz[u] = ld_x(&w.p_z[q]);
                vA[u] = ld_x(&w.p_mmA[q]);
                vB[u] = ld_x(&w.p_mmB[q]);
            }
#pragma unroll
            for (int u = 0; u < U; u++) {
                mm_merge((uint32_t)vA[u], (uint32_t)vB[u], lo3, hi3);   // a repeated row changes nothing
                if (b0 + u * ng >= st.gx) continue;
                sd += vsd[u]; sdn += vsdn[u]; z += vz[u];
            }
        }
    tSd[t] = sd; tZ[t] = z; tSdn[t] = sdn;
#pragma unroll
    for (int k = 0; k < 3; k++) { tMM[2 * k * kNT + t] = lo3[k]; tMM[(2 * k + 1) * kNT + t] = hi3[k]; }
    __syncthreads();
    if (t < CS) {
        for (int g2 = 1; g2 < ng; g2++) {
            const int i = g2 * CS + t;
            sd += tSd[i]; z += tZ[i]; sdn += tSdn[i];
#pragma unroll
            for (int k = 0; k < 3; k++) {
                lo3[k] = min(lo3[k], tMM[2 * k * kNT + i]);
                hi3[k] = max(hi3[k], tMM[(2 * k + 1) * kNT + i]);
            }
        }
        int mm[6];
#pragma unroll
        for (int k = 0; k < 3; k++) { mm[2 * k] = lo3[k] - 128; mm[2 * k + 1] = hi3[k] - 128; }   // empty: lo > hi
        const int64_t c = cb + t;
        w.sd[c] = sd; w.sdn[c] = sdn; w.Z[c] = z;
#pragma unroll
        for (int k = 0; k < 6; k++) w.mm[c * 6 + k] = mm[k];
        o.dbeta[c] = sd;
        o.dgamma[c] = sdn;
        // the channel totals, in the slots of group 0, for the candidate threads
        tSd[t] = sd; tZ[t] = z; tSdn[t] = sdn;
#pragma unroll
        for (int k = 0; k < 6; k++) tMM[k * kNT + t] = mm[k];
    }
    __syncthreads();
}

// largest of the slice's per-channel values in tCand (6 per channel) into
// *dst (kSentinelLo when none)
__device__ __forceinline__ void slice_cand_max(const int32_t* tCand, int n, int32_t* dst, int32_t* sh)
{
    int32_t m = kSentinelLo;
    for (int i = threadIdx.x; i < n; i += blockDim.x) m = max(m, tCand[i]);
    m = block_max_nt(m, sh);
    if (threadIdx.x == 0) *dst = m;
}

// stats tail (rounding E2).  Slice: the pass-1 sums, dgamma, dbeta and the
// largest |gamma_q delta| over its channels' sgn classes, into smaxF; the
// second pass takes E2's Scale from the largest over the slices.
__device__ __forceinline__ void bnb_round_tail1(uint32_t* lds, const Stream& st, const BwdWs& w, const Saved& sv,
                                                const BnCfg& cf, const BnbOut& o)
{
    bnb_tail_reduce1(lds, st, w, o);
    const int CS = st.CS, t = threadIdx.x;
    const Tail1Lds L(lds);
    __shared__ int32_t rb[kNT / 64];
    const int64_t cb = (int64_t)blockIdx.y * CS;
    int F = 0;
    if (t < CS) {
        int amax = 0;
        for (int k = 0; k < 3; k++) {
            const int lo = L.mm[2 * k * kNT + t], hi = L.mm[(2 * k + 1) * kNT + t];
            if (lo > hi) continue;                     // empty class
            amax = max(amax, max(lo < 0 ? -lo : lo, hi < 0 ? -hi : hi));
        }
        const int gq = o.gamma_q[cb + t];
        F = (gq < 0 ? -gq : gq) * amax;                // <= 128 * 128
    }
    F = block_max_nt(F, rb);
    if (t == 0) w.smaxF[blockIdx.y] = F;
}

// stats2 tail.  Slice: the pass-2 sums (sum f, sum f n_xhat) and each
// channel's bound on max|dx| (six candidates, as the exact tail); the largest
// goes to smax.  `lds` is stats2's x-hat table, no longer read.
__device__ __forceinline__ void bnb_round_tail2(uint32_t* lds, const Stream& st, const BwdWs& w,
                                                const Saved& sv, const BnCfg& cf, const BnbOut& o, int r2)
{
    const int CS = st.CS, ng = kNT / CS, t = threadIdx.x, ch = t % CS, grp = t / CS;
    long long* tSf = (long long*)lds;                   // [kNT]
    long long* tSfn = tSf + kNT;                        // [kNT]
    int32_t* tCand = (int32_t*)(tSfn + kNT);            // [6 * CS]
    __shared__ int32_t rb[kNT / 64];
    const int64_t cb = (int64_t)blockIdx.y * CS;
    long long sf = 0, sfn = 0;
    constexpr int U = 8;                    // partial rows whose loads are in flight together
    if (grp < ng)
        for (int b0 = grp; b0 < st.gx; b0 += U * ng) {
            long long vf[U], vn[U];
#pragma unroll
            for (int u = 0; u < U; u++) {
                const int b = b0 + u * ng;
                const int64_t q = (int64_t)(b < st.gx ? b : b0) * st.C + cb + ch;
                vf[u] = ld_x(&w.p_sf[q]);
                vn[u] = ld_x(&w.p_sfn[q]);
            }
#pragma unroll
            for (int u = 0; u < U; u++)
                if (b0 + u * ng < st.gx) { sf += vf[u]; sfn += vn[u]; }
        }
    tSf[t] = sf; tSfn[t] = sfn;
    __syncthreads();
    if (t < CS) {
        for (int g2 = 1; g2 < ng; g2++) { sf += tSf[g2 * CS + t]; sfn += tSfn[g2 * CS + t]; }
        w.sf[cb + t] = sf; w.sfn[cb + t] = sfn;
        tSf[t] = sf; tSfn[t] = sfn;                     // only thread t reads slot t above
    }
    __syncthreads();
    if (t < 6 * CS) {
        const int cl = t / 6, k = t % 6;                // channel of the slice; class k / 2, low / high
        const int64_t c = cb + cl;
        const int lo = w.mm[c * 6 + (k & ~1)], hi = w.mm[c * 6 + (k | 1)];
        int best = kSentinelLo;
        if (lo <= hi) {
            const int gq = o.gamma_q[c];
            const BnbChan e = bnb_chan_exps(r2, *o.dy_exp, sv, cf);
            const i128 M = st.M;
            const int64_t f = sq_code((int64_t)gq * ((k & 1) ? hi : lo), e.r2, cf.k_E2);
            const i128 B = bnb_bracket(f, (k >> 1) - 1, M, (i128)tSf[cl], (i128)tSfn[cl], (i128)w.Z[c], e.e_xh);
            if (B != 0) best = ceil_pow2_exp128(abs128(B), (i128)sv.den[c] * M * M) + e.Ebase;
        }
        tCand[t] = best;
    }
    __syncthreads();
    slice_cand_max(tCand, 6 * CS, w.smax + blockIdx.y, rb);
}

// Exact E2 (k_E2 >= 15), one block per channel and one thread per masked
// error code: the channel's totals from the streaming blocks' partials
// (dbeta, dgamma), its bound on E1's exponent (the largest over its six
// per-class extremes; xhat and the bracket are linear in the code, so the
// extremes bound every code the channel's data holds), and its dx values at
// that bound: Q = floor(B 2^S / D) with S one more than the shift of the
// channel's own bound, for the (class, code) pairs inside the channel's
// per-class ranges (zero elsewhere: the output pass never looks them up).
// |Q| <= 2^k_E1 + 1 there, so int16 holds it; the output pass rounds Q by
// the gap between the largest bound and the channel's into the final code
// (half-up rounding of floor(x) by 2^g + 1 equals that of x).
__global__ __launch_bounds__(256) void k_bnb_chan_exact(int64_t Mrows, int gx, int CS, BwdWs w, Saved sv,
                                                        BnCfg cf, BnbOut o)
{
    __shared__ int32_t r_sd[4], r_z[4], r_lo[4][3], r_hi[4][3], r_cand;
    __shared__ long long r_sdn[4];
    const int c = blockIdx.x, t = threadIdx.x, lane = t & 63, wv = t >> 6;
    int sd = 0, z = 0;
    long long sdn = 0;
    int lo3[3] = {255, 255, 255}, hi3[3] = {0, 0, 0};       // byte-coded extremes (empty: lo > hi)
    const int sy = c / CS, sc = c - sy * CS;                  // slice, channel within it
    for (int b = t; b < gx; b += blockDim.x) {
        const int64_t q = ((int64_t)sy * gx + b) * CS + sc;
        sd += w.p_sd[q];
        sdn += w.p_sdn[q];
        z += w.p_z[q];
        mm_merge((uint32_t)w.p_mmA[q], (uint32_t)w.p_mmB[q], lo3, hi3);
    }
    for (int off = 32; off > 0; off >>= 1) {
        sd += __shfl_xor(sd, off, 64);
        z += __shfl_xor(z, off, 64);
        sdn += __shfl_xor(sdn, off, 64);
#pragma unroll
        for (int k = 0; k < 3; k++) {
            lo3[k] = min(lo3[k], __shfl_xor(lo3[k], off, 64));
            hi3[k] = max(hi3[k], __shfl_xor(hi3[k], off, 64));
        }
    }
    if (lane == 0) {
        r_sd[wv] = sd; r_z[wv] = z; r_sdn[wv] = sdn;
#pragma unroll
        for (int k = 0; k < 3; k++) { r_lo[wv][k] = lo3[k]; r_hi[wv][k] = hi3[k]; }
    }
    __syncthreads();
    sd = (r_sd[0] + r_sd[1]) + (r_sd[2] + r_sd[3]);
    z = (r_z[0] + r_z[1]) + (r_z[2] + r_z[3]);
    sdn = (r_sdn[0] + r_sdn[1]) + (r_sdn[2] + r_sdn[3]);
    int mm[6];
#pragma unroll
    for (int k = 0; k < 3; k++) {
        mm[2 * k] = min(min(r_lo[0][k], r_lo[1][k]), min(r_lo[2][k], r_lo[3][k])) - 128;
        mm[2 * k + 1] = max(max(r_hi[0][k], r_hi[1][k]), max(r_hi[2][k], r_hi[3][k])) - 128;
    }
    if (t == 0) {
        o.dbeta[c] = sd;
        o.dgamma[c] = sdn;
    }
    const int gq = o.gamma_q[c];
    const int e_xh = sv.hdr[0] - (cf.k_xhat - 1);
    const int e_sig = 2 - cf.k_sigma, e_g = 2 - cf.k_gamma;
    const int Ebase = *o.dy_exp + e_g - e_sig + (e_xh < 0 ? e_xh : 0);
    const i128 M = Mrows;
    const i128 Dd = (i128)sv.den[c] * M * M;
    const i128 Sf = (i128)gq * sd, T = (i128)gq * sdn, Z = z;
    // the six per-class candidates (threads 0..5 of wave 0), their max
    if (wv == 0) {
        int cand = kSentinelLo;
        if (t < 6) {
            const int lo = mm[t & ~1], hi = mm[t | 1];
            if (lo <= hi) {
                const int64_t f = clamp_k((int64_t)gq * ((t & 1) ? hi : lo), cf.k_E2);
                const i128 B = bnb_bracket(f, (t >> 1) - 1, M, Sf, T, Z, e_xh);
                if (B != 0) cand = ceil_pow2_exp128(abs128(B), Dd) + Ebase;
            }
        }
        for (int off = 4; off > 0; off >>= 1) cand = max(cand, __shfl_xor(cand, off, 64));
        if (t == 0) {
            r_cand = cand;
            w.cbnd[c] = cand;
        }
    }
    __syncthreads();
    const int bc = r_cand;
    const int d = t - 128;
    const int S = Ebase + (cf.k_E1 - 1) - bc + 1;
    for (int k = 0; k < 3; k++) {
        int16_t q = 0;
        if (bc != kSentinelLo && d >= mm[2 * k] && d <= mm[2 * k + 1] && d >= -127) {
            const int64_t f = clamp_k((int64_t)gq * d, cf.k_E2);
            const i128 B = bnb_bracket(f, k - 1, M, Sf, T, Z, e_xh);
            i128 Q = S >= 0 ? floordiv128(B << S, Dd) : floordiv128(B, Dd << -S);
            Q = Q > 32767 ? 32767 : (Q < -32767 ? -32767 : Q);
            q = (int16_t)Q;
        }
        w.lutq[((int64_t)c * 3 + k) * 256 + t] = q;
    }
}

// Output pass: dx code = lut[c][sgn class][masked delta].  A per-(channel,
// code) entry gives the offset of the channel's class row in the block's LDS
// copy of the tables (bits 16..31) and the ReLU mask byte (bits 0..7), so each
// element costs two LDS reads and a handful of ALU operations.
// Exact E2: every block first takes E1's exponent from the channels' bounds
// (block (0, 0) writes it and the parameter-gradient exponents) and rounds
// its channels' staged values into the codes.
__global__ __launch_bounds__(1024) void k_bnb_apply(const int8_t* __restrict__ dy,
                                                   const int8_t* __restrict__ x,
                                                   int8_t* __restrict__ dx, Stream st, BwdWs w,
                                                   Saved sv, BnCfg cf, BnbOut o, int32_t exact)
{
    __shared__ __attribute__((aligned(16))) int8_t lut[64 * 3 * kRowB];
    __shared__ __attribute__((aligned(16))) uint32_t tab[64 * kRowW];
    __shared__ int32_t rb[kNT / 64];
    const int relu = cf.relu;
    const int64_t cbase = (int64_t)blockIdx.y * st.CS;
    if (exact) {
        int bdx = kSentinelLo;
        for (int i = threadIdx.x; i < st.C; i += kNT) bdx = max(bdx, w.cbnd[i]);
        bdx = block_max_nt(bdx, rb);
        if (bdx == kSentinelLo) bdx = 0;
        if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) {
            *o.dx_exp = bdx - (cf.k_E1 - 1);
            bnb_exps_out(sv, cf, o);
        }
        const short lim = (short)((1 << (cf.k_E1 - 1)) - 1);
        const int16_t* src = w.lutq + cbase * 768;
        for (int v = threadIdx.x; v < st.CS * 96; v += kNT) {      // eight values per step, two per op
            const int i0 = v * 8, row = i0 >> 8, col = i0 & 255;
            const int bc = w.cbnd[cbase + row / 3];
            const short sh = (short)(bc == kSentinelLo ? 15 : min(bdx - bc, 15));
            const int4 q = *(const int4*)(src + i0);
            const int qw[4] = {q.x, q.y, q.z, q.w};
            uint32_t ow[2] = {0, 0};
#pragma unroll
            for (int h = 0; h < 4; h++) {
                short2v qv = __builtin_bit_cast(short2v, qw[h]);
                qv = ((qv >> sh) + (short)1) >> (short)1;
                qv = qv > lim ? lim : qv;
                qv = qv < (short)-lim ? (short)-lim : qv;
                const uint32_t b = (uint32_t)(uint16_t)qv.x & 0xffu | ((uint32_t)(uint16_t)qv.y & 0xffu) << 8;
                ow[h >> 1] |= b << (16 * (h & 1));
            }
            *(uint32_t*)(lut + row * kRowB + col) = ow[0];
            *(uint32_t*)(lut + row * kRowB + col + 4) = ow[1];
        }
    } else {
        copy_rows_to_lds<64 * 3 * 16 / kNT>(lut, w.lut + cbase * 768, st.CS * 3);
    }
    load_bwd_tab(tab, sv.btab + cbase * 256, st.CS, relu, true);
    __syncthreads();
    int g, rsub;
    if (!stream_lane(st, g, rsub)) return;
    const int c0 = (int)cbase + g * 4;
    const uint32_t* tb = tab + g * 4 * kRowW;
    const int64_t step = (int64_t)gridDim.x * st.rpi;
    auto elem = [&](uint32_t wx, uint32_t wd) {
        uint32_t ow = 0;
#pragma unroll
        for (int i = 0; i < 4; i++) {
            const uint32_t e = tb[i * kRowW + ((wx >> (8 * i)) & 0xff)];
            const int idx = (int)(e >> 16) + (sbyte(wd, i) & (int)(int8_t)(e & 0xff));
            ow |= (uint32_t)(uint8_t)lut[idx] << (8 * i);
        }
        return ow;
    };
    // full groups of U rows with the next group's loads in flight, then the rest
    constexpr int U = 4;
    int64_t r = (int64_t)blockIdx.x * st.rpi + rsub;
    const int64_t full_end = st.M - (U - 1) * step;
    uint32_t vx[U], vd[U], nx[U], nd[U];
    auto load = [&](int64_t r0, uint32_t* ax, uint32_t* ad) {
#pragma unroll
        for (int u = 0; u < U; u++) {
            ax[u] = *(const uint32_t*)(x + (r0 + u * step) * st.C + c0);
            ad[u] = *(const uint32_t*)(dy + (r0 + u * step) * st.C + c0);
        }
    };
    if (r < full_end) load(r, vx, vd);
    while (r < full_end) {
        const int64_t rn = r + U * step;
        if (rn < full_end) load(rn, nx, nd);
#pragma unroll
        for (int u = 0; u < U; u++) *(uint32_t*)(dx + (r + u * step) * st.C + c0) = elem(vx[u], vd[u]);
#pragma unroll
        for (int u = 0; u < U; u++) { vx[u] = nx[u]; vd[u] = nd[u]; }
        r = rn;
    }
    for (; r < st.M; r += step)
        *(uint32_t*)(dx + r * st.C + c0) =
            elem(*(const uint32_t*)(x + r * st.C + c0), *(const uint32_t*)(dy + r * st.C + c0));
}

bool cfg_ok(const iseg_bn_cfg* c)
{
    if (!c) return false;
    auto in = [](int v, int lo, int hi) { return v >= lo && v <= hi; };
    return in(c->k_mu, 2, 16) && in(c->k_sigma, 2, 16) && in(c->k_xhat, 2, 16) &&
           in(c->k_gamma, 2, 8) && in(c->k_beta, 2, 8) && in(c->k_A, 2, 8) && in(c->k_E1, 2, 8) &&
           in(c->k_E2, 2, 16) && in(c->eps_code, 0, 1 << 15) && (c->relu == 0 || c->relu == 1);
}

// forward statistics geometry; the 4-channel-lane variant has the most
// blocks, so it sizes the workspace for both
Stream fwd_stats_stream(int64_t M, int64_t C, int cs, bool v16)
{
    return make_stream(M, C, cs, v16 && ISEG_BNF_STATS_CPL == 16 ? 16 : 4, 4, kMaxBlocks);
}

bool shape_ok(int64_t M, int64_t C) { return M >= 1 && C >= 4 && M <= ((int64_t)1 << 22) && C <= (1 << 16); }

}  // namespace

// ---------------------------------------------------------------------------
// C ABI
// ---------------------------------------------------------------------------
extern "C" size_t iseg_bn_saved_bytes(int64_t C) { return C > 0 ? saved_bytes(C) : 0; }

extern "C" size_t iseg_bn_fwd_ws(int64_t M, int64_t C)
{
    int cs = pick_cs(C, 128);
    if (!shape_ok(M, C) || !cs) return 0;
    return fwd_ws_bytes(fwd_stats_stream(M, C, cs, false));
}

extern "C" size_t iseg_bn_bwd_ws(int64_t M, int64_t C)
{
    int cs = pick_cs(C, 64);
    if (!shape_ok(M, C) || !cs) return 0;
    return bwd_ws_bytes(make_stream(M, C, cs, 4, ISEG_BNB_ROWS, kMaxBlocks));
}

static int bn_fwd_impl(const int8_t* x, const int32_t* x_exp, int64_t M, int64_t C,
                       const int8_t* gamma_q, const int8_t* beta_q, const iseg_bn_cfg* cfg,
                       int8_t* y_out, int32_t* y_exp, void* saved,
                       void* ws, size_t ws_bytes, int32_t* dev_status, hipStream_t stream)
{
    if (M < 1 || C < 4) return ISEG_ERR_SHAPE;
    if (!shape_ok(M, C)) return ISEG_ERR_UNSUPPORTED;
    if (!x || !x_exp || !gamma_q || !beta_q || !y_out || !y_exp || !saved || !cfg_ok(cfg))
        return ISEG_ERR_ARG;
    int cs = pick_cs(C, 128);
    if (!cs || (((uintptr_t)x | (uintptr_t)y_out) & 3)) return ISEG_ERR_UNSUPPORTED;
    const bool v16 = cs % 16 == 0 && (((uintptr_t)x | (uintptr_t)y_out) & 15) == 0;
    const bool s16 = v16 && ISEG_BNF_STATS_CPL == 16;
    Stream st = fwd_stats_stream(M, C, cs, v16);
    if (!ws || ws_bytes < fwd_ws_bytes(fwd_stats_stream(M, C, cs, false))) return ISEG_ERR_WORKSPACE;
    BnCfg cf = to_cfg(cfg);
    Saved sv = saved_map(saved, C);
    FwdWs w = fwd_ws_map(ws, st);
    dim3 sg = stream_grid(st);
    dim3 cb((unsigned)C);
    if (s16)
        ISEG_TIMED_LAUNCH(ISEG_KID_BN_FWD_STATS1, stream, k_bnf_stats1<16>, sg, dim3(kNT), 0, stream, x, st, w);
    else
        ISEG_TIMED_LAUNCH(ISEG_KID_BN_FWD_STATS1, stream, k_bnf_stats1<4>, sg, dim3(kNT), 0, stream, x, st, w);
    if (s16)
        ISEG_TIMED_LAUNCH(ISEG_KID_BN_FWD_STATS2, stream, k_bnf_stats2<16>, sg, dim3(kNT), 0, stream, x, x_exp,
                          st, w, sv, cf, dev_status);
    else
        ISEG_TIMED_LAUNCH(ISEG_KID_BN_FWD_STATS2, stream, k_bnf_stats2<4>, sg, dim3(kNT), 0, stream, x, x_exp,
                          st, w, sv, cf, dev_status);
    hipLaunchKernelGGL(k_bnf_fin2, cb, dim3(256), 0, stream, x_exp, (int)sg.y, w, sv, cf, gamma_q, beta_q);
    if (v16) {
        Stream a16 = make_stream(M, C, cs, 16, 4, kMaxBlocks);
        ISEG_TIMED_LAUNCH(ISEG_KID_BN_FWD_APPLY, stream, k_bnf_apply<16>, stream_grid(a16), dim3(kNT), 0,
                          stream, x, y_out, a16, sv, w, cf, x_exp, gamma_q, beta_q, y_exp);
    } else {
        Stream s4 = make_stream(M, C, cs, 4, 4, kMaxBlocks);
        ISEG_TIMED_LAUNCH(ISEG_KID_BN_FWD_APPLY, stream, k_bnf_apply<4>, stream_grid(s4), dim3(kNT), 0, stream,
                          x, y_out, s4, sv, w, cf, x_exp, gamma_q, beta_q, y_exp);
    }
    return launch_ok();
}

extern "C" int iseg_bn_fwd(const int8_t* x, const int32_t* x_exp, int64_t M, int64_t C,
                           const int8_t* gamma_q, const int8_t* beta_q, const iseg_bn_cfg* cfg,
                           int8_t* y_out, int32_t* y_exp, void* saved,
                           void* ws, size_t ws_bytes, int32_t* dev_status, hipStream_t stream)
{
    return bn_fwd_impl(x, x_exp, M, C, gamma_q, beta_q, cfg, y_out, y_exp, saved, ws, ws_bytes, dev_status,
                       stream);
}

// ---------------------------------------------------------------------------
// iseg_bn_fwd_noalloc: the same forward with its workspace in a static device
// array (one copy per GPU, held until the process ends) instead of a caller
// buffer.  In host code `scratch` names a host-side stand-in, not device
// memory: its device address is looked up once per device with
// hipGetSymbolAddress (with that device current) and only that address is
// passed to the kernels.  The array starts at zero and every call leaves
// the forward's arrival counters at zero; the rest of the workspace is
// written before it is read within a call, so nothing needs clearing between
// calls.
// ---------------------------------------------------------------------------
namespace {
constexpr size_t kBnScratchBytes = (size_t)1 << 20;
constexpr int kScratchDevices = 64;
__device__ __align__(256) unsigned char scratch[kBnScratchBytes];
std::mutex g_scratch_mu;
void* g_scratch_ptr[kScratchDevices] = {};
}  // namespace

static void* bn_scratch_ptr()
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kScratchDevices) return nullptr;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
        g_scratch_ptr[dev] = p;
    }
    return g_scratch_ptr[dev];
}

extern "C" size_t iseg_bn_fwd_noalloc_max_bytes(void) { return kBnScratchBytes; }

extern "C" int iseg_bn_fwd_noalloc(const int8_t* x, const int32_t* x_exp, int64_t M, int64_t C,
                                   const int8_t* gamma_q, const int8_t* beta_q, const iseg_bn_cfg* cfg,
                                   int8_t* y_out, int32_t* y_exp, void* saved, int32_t* dev_status,
                                   hipStream_t stream)
{
    const size_t need = iseg_bn_fwd_ws(M, C);
    if (need == 0) return M < 1 || C < 4 ? ISEG_ERR_SHAPE : ISEG_ERR_UNSUPPORTED;
    if (need > kBnScratchBytes) return ISEG_ERR_WORKSPACE;
    void* ws = bn_scratch_ptr();
    if (!ws) return ISEG_ERR_DEVICE;
    return bn_fwd_impl(x, x_exp, M, C, gamma_q, beta_q, cfg, y_out, y_exp, saved, ws, kBnScratchBytes,
                       dev_status, stream);
}

extern "C" int iseg_bn_bwd(const int8_t* dy, const int32_t* dy_exp, const int8_t* x,
                           int64_t M, int64_t C, const int8_t* gamma_q, const iseg_bn_cfg* cfg,
                           const void* saved, int8_t* dx_out, int32_t* dx_exp,
                           int64_t* dgamma, int64_t* dbeta, int32_t* dgamma_exp, int32_t* dbeta_exp,
                           void* ws, size_t ws_bytes, int32_t* dev_status, hipStream_t stream)
{
    if (M < 1 || C < 4) return ISEG_ERR_SHAPE;
    if (!shape_ok(M, C)) return ISEG_ERR_UNSUPPORTED;
    if (!dy || !dy_exp || !x || !gamma_q || !saved || !dx_out || !dx_exp || !dgamma || !dbeta ||
        !dgamma_exp || !dbeta_exp || !cfg_ok(cfg))
        return ISEG_ERR_ARG;
    int cs = pick_cs(C, 64);
    if (!cs || (((uintptr_t)x | (uintptr_t)dy | (uintptr_t)dx_out) & 3)) return ISEG_ERR_UNSUPPORTED;
    Stream st = make_stream(M, C, cs, 4, ISEG_BNB_ROWS, kMaxBlocks);
    if (!ws || ws_bytes < bwd_ws_bytes(st)) return ISEG_ERR_WORKSPACE;
    BnCfg cf = to_cfg(cfg);
    Saved sv = saved_map((void*)saved, C);
    BwdWs w = bwd_ws_map(ws, st);
    dim3 sg = stream_grid(st);
    dim3 cb((unsigned)C);
    // E2 = SQ(gamma delta, k_E2) is exact when |gamma delta| <= 127^2 < 2^(k_E2-1)
    const int exact_e2 = cf.k_E2 >= 15;
    const BnbOut out{dy_exp, gamma_q, dgamma, dbeta, dgamma_exp, dbeta_exp, dx_exp, dev_status};
    if (exact_e2) {
        ISEG_TIMED_LAUNCH(ISEG_KID_BN_BWD_STATS, stream, k_bnb_stats<1>, sg, dim3(kNT), 0, stream, dy, x, st, w,
                          sv, cf, out);
        hipLaunchKernelGGL(k_bnb_chan_exact, cb, dim3(256), 0, stream, M, (int)st.gx, (int)st.CS, w, sv, cf, out);
    } else {
        ISEG_TIMED_LAUNCH(ISEG_KID_BN_BWD_STATS, stream, k_bnb_stats<2>, sg, dim3(kNT), 0, stream, dy, x, st,
                          w, sv, cf, out);
        hipLaunchKernelGGL(k_bnb_stats2, sg, dim3(kNT), 0, stream, dy, x, st, w, sv, cf, out);
        hipLaunchKernelGGL(k_bnb_lut, cb, dim3(256), 0, stream, M, (int)sg.y, w, sv, cf, out);
    }
    // the output pass needs no partials: its grid holds more rows per lane
    const Stream sa = make_stream(M, C, cs, 4, 8, kMaxBlocks);
    ISEG_TIMED_LAUNCH(ISEG_KID_BN_BWD_APPLY, stream, k_bnb_apply, stream_grid(sa), dim3(kNT), 0, stream, dy, x,
                      dx_out, sa, w, sv, cf, out, exact_e2);
    return launch_ok();
}

// ---------------------------------------------------------------------------
// Inference with the frozen state of a calibration forward (the state that
// iseg_bn_fwd saved): the per-(channel, code) A table, built from that pass's
// n_mu, denominator and the fixed steps of Q_xhat and Q_A, is applied to new
// inputs.  A wide input (the raw int32 sums of a conv) first goes to the
// calibration's Z grid with a fixed-step quantizer (half-up, clipped to 8
// bits): the requant, L1BN, ReLU and Q_A of a layer in one pass.
// ---------------------------------------------------------------------------
namespace {
template <bool WIDE>
__global__ __launch_bounds__(256) void k_bn_infer(const void* __restrict__ in, const int32_t* in_exp,
                                                  const int32_t* w_exp, int64_t n4, int32_t C, Saved sv,
                                                  int8_t* __restrict__ out, int32_t* out_exp,
                                                  int32_t* dev_status)
{
    const int32_t ez = sv.hdr[3];
    const int32_t es = *in_exp + (WIDE ? *w_exp : 0);
    const int r = ez - es;                 // Z = sums 2^-r on the calibration's grid
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        *out_exp = sv.hdr[2];
        if (!WIDE && r != 0) set_status(dev_status, ISEG_DEV_RANGE);   // codes on another grid
    }
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) {
        const int c0 = (int)((i * 4) % C);
        int z[4];
        if (WIDE) {
            const int4 v = ((const int4*)in)[i];
            const int s[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int j = 0; j < 4; j++) {
                int64_t q;
                if (r > 0) q = ((int64_t)s[j] + ((int64_t)1 << (r - 1))) >> r;
                else if (r >= -32) q = (int64_t)s[j] * ((int64_t)1 << -r);
                else q = s[j] > 0 ? 128 : (s[j] < 0 ? -128 : 0);
                z[j] = (int)clamp_k(q, 8);
            }
        } else {
            const uint32_t v = ((const uint32_t*)in)[i];
#pragma unroll
            for (int j = 0; j < 4; j++) z[j] = (int)(int8_t)(v >> (8 * j));
        }
        uint32_t o = 0;
#pragma unroll
        for (int j = 0; j < 4; j++)
            o |= (uint32_t)(uint8_t)sv.acode[(int64_t)(c0 + j) * 256 + z[j] + 128] << (8 * j);
        ((uint32_t*)out)[i] = o;
    }
}
}  // namespace

extern "C" int iseg_bn_infer(const int8_t* z, const int32_t* z_exp, int64_t M, int64_t C, const void* saved,
                             int8_t* a_out, int32_t* a_exp, int32_t* dev_status, hipStream_t stream)
{
    if (M < 1 || C < 4) return ISEG_ERR_SHAPE;
    if (!shape_ok(M, C) || C % 4) return ISEG_ERR_UNSUPPORTED;
    if (!z || !z_exp || !saved || !a_out || !a_exp) return ISEG_ERR_ARG;
    if (((uintptr_t)z | (uintptr_t)a_out) & 3) return ISEG_ERR_UNSUPPORTED;
    const Saved sv = saved_map((void*)saved, C);
    const int64_t n4 = M * C / 4;
    hipLaunchKernelGGL(k_bn_infer<false>, dim3(grid_for(n4, 256 * 4, 4096)), dim3(256), 0, stream, z, z_exp,
                       z_exp, n4, (int32_t)C, sv, a_out, a_exp, dev_status);
    return launch_ok();
}

extern "C" size_t iseg_conv_bn_infer_ws(const iseg_conv_geom* g)
{
    const size_t cw = iseg_conv_fwd_ws(g, ISEG_OUT_RAW);
    if (!cw || !g) return 0;
    const int64_t P = (g->H + 2 * g->pad_h - g->dil_h * (g->R - 1) - 1) / g->stride_h + 1;
    const int64_t Q = (g->W + 2 * g->pad_w - g->dil_w * (g->S - 1) - 1) / g->stride_w + 1;
    return align256((size_t)(g->N * P * Q * g->K) * 4) + cw;
}

extern "C" int iseg_conv_bn_infer(const int8_t* x, const int32_t* x_exp, const int8_t* w, const int32_t* w_exp,
                                  const iseg_conv_geom* g, const void* saved, int8_t* a_out, int32_t* a_exp,
                                  void* ws, size_t ws_bytes, int32_t* dev_status, hipStream_t stream)
{
    if (!g || !saved || !a_out || !a_exp || !x_exp || !w_exp) return ISEG_ERR_ARG;
    const size_t need = iseg_conv_bn_infer_ws(g);
    if (!need) return ISEG_ERR_SHAPE;
    if (!ws || ws_bytes < need) return ISEG_ERR_WORKSPACE;
    const int64_t P = (g->H + 2 * g->pad_h - g->dil_h * (g->R - 1) - 1) / g->stride_h + 1;
    const int64_t Q = (g->W + 2 * g->pad_w - g->dil_w * (g->S - 1) - 1) / g->stride_w + 1;
    const int64_t M = g->N * P * Q, C = g->K;
    if (M < 1 || C < 4) return ISEG_ERR_SHAPE;
    if (!shape_ok(M, C) || C % 4 || ((uintptr_t)a_out & 3)) return ISEG_ERR_UNSUPPORTED;
    int32_t* sums = (int32_t*)ws;
    char* cws = (char*)ws + align256((size_t)(M * C) * 4);
    // the sums' own exponent slot: the conv writes x_exp + w_exp there; the pass reads both inputs' exponents
    int32_t* sexp = (int32_t*)a_exp;
    int rc = iseg_conv_fwd(x, x_exp, w, w_exp, g, ISEG_OUT_RAW, sums, sexp, cws, ws_bytes - (cws - (char*)ws),
                           dev_status, stream);
    if (rc) return rc;
    const Saved sv = saved_map((void*)saved, C);
    const int64_t n4 = M * C / 4;
    hipLaunchKernelGGL(k_bn_infer<true>, dim3(grid_for(n4, 256 * 4, 4096)), dim3(256), 0, stream, sums, x_exp,
                       w_exp, n4, (int32_t)C, sv, a_out, a_exp, dev_status);
    return launch_ok();
}
