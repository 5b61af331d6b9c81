// quant.hip -- the quantizers (Eq. 2 UQ, Eq. 3-4 SQ, Eq. 5-6 RQ), the update
// and weight quantizers (Eq. 19, Eq. 8) and the shared requant machinery.
//
// All of these are bandwidth-bound streams: one pass computes max|x| with a
// wave reduction and one atomicMax per block, a second pass turns elements
// into codes with 16-byte vector loads where the dtype allows.
#include "iseg_common.h"

// ---------------------------------------------------------------------------
// fill / absmax
// ---------------------------------------------------------------------------
__global__ void k_fill_u32(uint32_t* p, int64_t n, uint32_t v)
{
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

int launch_fill_u32(void* p, int64_t n_words, uint32_t v, hipStream_t s)
{
    if (n_words <= 0) return ISEG_OK;
    hipLaunchKernelGGL(k_fill_u32, dim3(grid_for(n_words, 256, 1024)), dim3(256), 0, s,
                       (uint32_t*)p, n_words, v);
    return launch_ok();
}

__device__ __forceinline__ uint64_t uabs64(int64_t v)
{
    return v < 0 ? (uint64_t)0 - (uint64_t)v : (uint64_t)v;
}

template <typename T>
__global__ __launch_bounds__(256) void k_absmax_scalar(const T* __restrict__ in, int64_t n,
                                                       unsigned long long* maxp)
{
    uint64_t m = 0;
    for (int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; j < n;
         j += (int64_t)gridDim.x * blockDim.x) {
        uint64_t a = uabs64((int64_t)in[j]);
        m = a > m ? a : m;
    }
    block_atomic_max_u64(m, maxp);
}

// int32 input, 16-byte aligned
template <typename T>
__global__ __launch_bounds__(256) void k_absmax(const T* __restrict__ in, int64_t n,
                                                unsigned long long* maxp)
{
    uint64_t m = 0;
    int64_t stride = (int64_t)gridDim.x * blockDim.x;
    int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (sizeof(T) == 4) {
        // 4 elements per step through int4 loads on the aligned body
        const int4* v4 = (const int4*)in;
        int64_t n4 = n >> 2;
        for (int64_t j = i; j < n4; j += stride) {
            int4 v = v4[j];
            uint64_t a = uabs64(v.x), b = uabs64(v.y), c = uabs64(v.z), d = uabs64(v.w);
            a = a > b ? a : b;
            c = c > d ? c : d;
            a = a > c ? a : c;
            m = a > m ? a : m;
        }
        for (int64_t j = (n4 << 2) + i; j < n; j += stride) {
            uint64_t a = uabs64((int64_t)in[j]);
            m = a > m ? a : m;
        }
    } else {
        for (int64_t j = i; j < n; j += stride) {
            uint64_t a = uabs64((int64_t)in[j]);
            m = a > m ? a : m;
        }
    }
    block_atomic_max_u64(m, maxp);
}

int launch_absmax(const void* in, int in_dtype, int64_t n, unsigned long long* maxp,
                  int32_t*, hipStream_t s)
{
    if (n <= 0) return ISEG_OK;
    if (in_dtype == ISEG_I32 && ((uintptr_t)in & 15) == 0)
        hipLaunchKernelGGL(k_absmax<int32_t>, dim3(grid_for(n, 256 * 16, 2048)), dim3(256), 0, s,
                           (const int32_t*)in, n, maxp);
    else if (in_dtype == ISEG_I32)
        hipLaunchKernelGGL(k_absmax_scalar<int32_t>, dim3(grid_for(n, 256 * 8, 2048)), dim3(256), 0, s,
                           (const int32_t*)in, n, maxp);
    else
        hipLaunchKernelGGL(k_absmax_scalar<int64_t>, dim3(grid_for(n, 256 * 8, 2048)), dim3(256), 0, s,
                           (const int64_t*)in, n, maxp);
    return launch_ok();
}

__global__ __launch_bounds__(1024) void k_reduce_max(const uint64_t* __restrict__ part, int64_t n,
                                                     unsigned long long* maxp)
{
    const uint64_t m = reduce_partials_u64(part, n);
    if (threadIdx.x == 0) *maxp = m;
}

int launch_reduce_max(const uint64_t* part, int64_t n, unsigned long long* maxp, hipStream_t s)
{
    hipLaunchKernelGGL(k_reduce_max, dim3(1), dim3(1024), 0, s, part, n, maxp);
    return launch_ok();
}

// ---------------------------------------------------------------------------
// requant apply: SQ half-up or RQ stochastic with r = bitlen(max) - (bits-1)
// ---------------------------------------------------------------------------
struct RqArgs {
    int64_t n;
    const int32_t* exp_a;
    const int32_t* exp_b;
    int32_t exp_add;
    int32_t bits, stochastic, keep_scale;
    uint64_t seed;
    uint32_t tensor_id, step;
    int32_t* out_exp;
    const unsigned long long* maxp;
    const uint64_t* part;
    int64_t nparts;
};

// the tensor max: from *maxp, or reduced by this block from the partials
__device__ __forceinline__ uint64_t rq_max(const RqArgs& a)
{
    return a.maxp ? (uint64_t)*a.maxp : reduce_partials_u64(a.part, a.nparts);
}

__device__ __forceinline__ int rq_shift(const RqArgs& a, uint64_t M)
{
    return M ? bitlen_u64(M) - (a.bits - 1) : 0;
}

__device__ __forceinline__ void rq_write_exp(const RqArgs& a, uint64_t M, int r)
{
    if (blockIdx.x == 0 && threadIdx.x == 0 && a.out_exp) {
        int32_t e = (a.exp_a ? *a.exp_a : 0) + (a.exp_b ? *a.exp_b : 0) + a.exp_add;
        *a.out_exp = a.keep_scale ? e + r : 1 - a.bits;
        (void)M;
    }
}

__device__ __forceinline__ int64_t rq_one(const RqArgs& a, int64_t q, int r, int64_t idx)
{
    if (a.stochastic && r > 0)
        return rq_code(q, r, a.bits, philox_draw(a.seed, a.tensor_id, a.step, (uint64_t)idx));
    return sq_code(q, r, a.bits);
}

// int32 -> int8, 16 elements per vector step
__global__ __launch_bounds__(256) void k_requant_i32_i8(const int32_t* __restrict__ in,
                                                        int8_t* __restrict__ out, RqArgs a)
{
    uint64_t M = rq_max(a);
    int r = rq_shift(a, M);
    rq_write_exp(a, M, r);
    int64_t stride = (int64_t)gridDim.x * blockDim.x;
    int64_t i0 = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    int64_t n16 = a.n >> 4;
    const int4* in4 = (const int4*)in;
    int4* out16 = (int4*)out;
    for (int64_t j = i0; j < n16; j += stride) {
        uint32_t w[4];
#pragma unroll
        for (int v = 0; v < 4; v++) {
            int4 q = in4[j * 4 + v];
            int64_t base = j * 16 + v * 4;
            uint32_t b0 = (uint8_t)rq_one(a, q.x, r, base + 0);
            uint32_t b1 = (uint8_t)rq_one(a, q.y, r, base + 1);
            uint32_t b2 = (uint8_t)rq_one(a, q.z, r, base + 2);
            uint32_t b3 = (uint8_t)rq_one(a, q.w, r, base + 3);
            w[v] = b0 | (b1 << 8) | (b2 << 16) | (b3 << 24);
        }
        out16[j] = make_int4((int)w[0], (int)w[1], (int)w[2], (int)w[3]);
    }
    for (int64_t j = (n16 << 4) + i0; j < a.n; j += stride)
        out[j] = (int8_t)rq_one(a, in[j], r, j);
}

template <typename TIn, typename TOut>
__global__ __launch_bounds__(256) void k_requant_generic(const TIn* __restrict__ in,
                                                         TOut* __restrict__ out, RqArgs a)
{
    uint64_t M = rq_max(a);
    int r = rq_shift(a, M);
    rq_write_exp(a, M, r);
    for (int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; j < a.n;
         j += (int64_t)gridDim.x * blockDim.x)
        out[j] = (TOut)rq_one(a, (int64_t)in[j], r, j);
}

int launch_requant_apply(const void* in, int in_dtype, int64_t n, const int32_t* exp_a,
                         const int32_t* exp_b, int32_t exp_add, int bits, int stochastic,
                         int keep_scale, uint64_t seed, uint32_t tensor_id, uint32_t step,
                         int out_dtype, void* out, int32_t* out_exp,
                         const unsigned long long* maxp, hipStream_t s, const uint64_t* part, int64_t nparts)
{
    RqArgs a;
    a.part = part; a.nparts = nparts;
    a.n = n; a.exp_a = exp_a; a.exp_b = exp_b; a.exp_add = exp_add;
    a.bits = bits; a.stochastic = stochastic; a.keep_scale = keep_scale;
    a.seed = seed; a.tensor_id = tensor_id; a.step = step;
    a.out_exp = out_exp; a.maxp = maxp;
    const unsigned cap = part ? 1024 : 4096;        // partials are read by every block
    bool aligned = (((uintptr_t)in | (uintptr_t)out) & 15) == 0;
    if (in_dtype == ISEG_I32 && out_dtype == ISEG_I8 && aligned)
        ISEG_TIMED_LAUNCH(ISEG_KID_REQUANT, s, k_requant_i32_i8, dim3(grid_for(n, 256 * 16, cap)), dim3(256), 0, s,
                           (const int32_t*)in, (int8_t*)out, a);
    else if (in_dtype == ISEG_I32 && out_dtype == ISEG_I8)
        ISEG_TIMED_LAUNCH(ISEG_KID_REQUANT, s, (k_requant_generic<int32_t, int8_t>), dim3(grid_for(n, 256, cap)),
                           dim3(256), 0, s, (const int32_t*)in, (int8_t*)out, a);
    else if (in_dtype == ISEG_I32 && out_dtype == ISEG_I16)
        ISEG_TIMED_LAUNCH(ISEG_KID_REQUANT, s, (k_requant_generic<int32_t, int16_t>), dim3(grid_for(n, 256, cap)),
                           dim3(256), 0, s, (const int32_t*)in, (int16_t*)out, a);
    else if (in_dtype == ISEG_I64 && out_dtype == ISEG_I8)
        ISEG_TIMED_LAUNCH(ISEG_KID_REQUANT, s, (k_requant_generic<int64_t, int8_t>), dim3(grid_for(n, 256, cap)),
                           dim3(256), 0, s, (const int64_t*)in, (int8_t*)out, a);
    else if (in_dtype == ISEG_I64 && out_dtype == ISEG_I16)
        ISEG_TIMED_LAUNCH(ISEG_KID_REQUANT, s, (k_requant_generic<int64_t, int16_t>), dim3(grid_for(n, 256, cap)),
                           dim3(256), 0, s, (const int64_t*)in, (int16_t*)out, a);
    else
        return ISEG_ERR_ARG;
    return launch_ok();
}

// SQ / RQ (Eq. 3-6) of the exact sum of S int32 partial tensors [S][n]
// (n % 4 == 0): four elements per thread step, every split's 16-byte load in
// flight together, the int64 sum formed in registers (never stored).
template <int S>
__global__ __launch_bounds__(256) void k_requant_splits_i8(const int32_t* __restrict__ part,
                                                           int8_t* __restrict__ out, RqArgs a)
{
    const uint64_t M = rq_max(a);
    const int r = rq_shift(a, M);
    rq_write_exp(a, M, r);
    const int64_t n4 = a.n >> 2;
    for (int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; j < n4; j += (int64_t)gridDim.x * blockDim.x) {
        int4 v[S];
#pragma unroll
        for (int k = 0; k < S; k++) v[k] = *(const int4*)(part + (int64_t)k * a.n + j * 4);
        int64_t s[4] = {0, 0, 0, 0};
#pragma unroll
        for (int k = 0; k < S; k++) { s[0] += v[k].x; s[1] += v[k].y; s[2] += v[k].z; s[3] += v[k].w; }
        uint32_t w = 0;
#pragma unroll
        for (int e = 0; e < 4; e++) w |= (uint32_t)(uint8_t)rq_one(a, s[e], r, j * 4 + e) << (8 * e);
        *(uint32_t*)(out + j * 4) = w;
    }
}

int launch_requant_splits(const int32_t* part, int splits, int64_t n, const int32_t* exp_a, const int32_t* exp_b,
                          int bits, int stochastic, int keep_scale, uint64_t seed, uint32_t tensor_id, uint32_t step,
                          int8_t* out, int32_t* out_exp, hipStream_t s, const uint64_t* pmax, int64_t npmax)
{
    if (splits < 1 || splits > 8 || n % 4 != 0 || (((uintptr_t)part) & 15) || (((uintptr_t)out) & 3))
        return ISEG_ERR_ARG;
    RqArgs a;
    a.part = pmax; a.nparts = npmax;
    a.n = n; a.exp_a = exp_a; a.exp_b = exp_b; a.exp_add = 0;
    a.bits = bits; a.stochastic = stochastic; a.keep_scale = keep_scale;
    a.seed = seed; a.tensor_id = tensor_id; a.step = step;
    a.out_exp = out_exp; a.maxp = nullptr;
    const dim3 grid(grid_for(n / 4, 256, 2048));
    switch (splits) {
#define ISEG_RQS(S) case S: ISEG_TIMED_LAUNCH(ISEG_KID_REQUANT, s, k_requant_splits_i8<S>, grid, dim3(256), 0, s, part, out, a); break;
    ISEG_RQS(1) ISEG_RQS(2) ISEG_RQS(3) ISEG_RQS(4) ISEG_RQS(5) ISEG_RQS(6) ISEG_RQS(7) ISEG_RQS(8)
#undef ISEG_RQS
    }
    return launch_ok();
}

// ---------------------------------------------------------------------------
// requant of int16-staged sums: element (m, n) of a [rows][cols] tensor holds
// floor(acc / 2^t) with t = tshift of its tile (rows in runs of tile_rows, or
// 2-D th x tw pixel tiles of an image when th > 0; tile_cols columns)
// and t <= r - 1 whenever t > 0, so the half-up code of acc by r is the half-up
// code of the staged value by r - t: ((y >> (r - 1 - t)) + 1) >> 1, clamped.
// 16 elements per thread step (cols % 16 == 0, all in one tile).
// ---------------------------------------------------------------------------
__device__ __forceinline__ int32_t clamp_k32(int32_t v, int k)
{
    const int32_t lim = (1 << (k - 1)) - 1;
    return v > lim ? lim : (v < -lim ? -lim : v);
}

__global__ __launch_bounds__(256) void k_requant_s16_i8(const int16_t* __restrict__ in,
                                                        const uint8_t* __restrict__ tshift, int64_t rows,
                                                        int32_t cols, StageMap sm, int8_t* __restrict__ out,
                                                        RqArgs a)
{
    const uint64_t M = rq_max(a);
    const int r = rq_shift(a, M);
    rq_write_exp(a, M, r);
    const int32_t cpr = cols >> 4;                        // 16-element chunks per row
    const int32_t tpr = cols / sm.tile_cols;              // column tiles
    const int64_t nch = rows * cpr;
    const int64_t hw = (int64_t)sm.Ho * sm.Wo;
    for (int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; j < nch;
         j += (int64_t)gridDim.x * blockDim.x) {
        const int64_t m = j / cpr;
        const int32_t n = (int32_t)(j - m * cpr) << 4;
        int64_t rt;                                       // row-tile index of row m
        if (sm.th == 0) {
            rt = m / sm.tile_rows;
        } else {                                          // 2-D pixel tiles of th x tw
            const int64_t img = m / hw;
            const int32_t rem = (int32_t)(m - img * hw);
            const int32_t oy = rem / sm.Wo, ox = rem - (rem / sm.Wo) * sm.Wo;
            rt = (img * sm.tiles_y + oy / sm.th) * sm.tiles_x + ox / sm.tw;
        }
        const int t = tshift[rt * tpr + n / sm.tile_cols];
        const int4 v0 = ((const int4*)in)[2 * j], v1 = ((const int4*)in)[2 * j + 1];
        const uint32_t h[8] = {(uint32_t)v0.x, (uint32_t)v0.y, (uint32_t)v0.z, (uint32_t)v0.w,
                               (uint32_t)v1.x, (uint32_t)v1.y, (uint32_t)v1.z, (uint32_t)v1.w};
        uint32_t w[4];
#pragma unroll
        for (int q = 0; q < 4; q++) {
            uint32_t o = 0;
#pragma unroll
            for (int b = 0; b < 4; b++) {
                const uint32_t hw = h[(4 * q + b) >> 1];
                const int32_t y = (int32_t)(int16_t)(((4 * q + b) & 1) ? (hw >> 16) : (hw & 0xffff));
                const int32_t c = r > 0 ? (((y >> (r - 1 - t)) + 1) >> 1) : (y << -r);
                o |= (uint32_t)(uint8_t)clamp_k32(c, a.bits) << (8 * b);
            }
            w[q] = o;
        }
        ((int4*)out)[j] = make_int4((int)w[0], (int)w[1], (int)w[2], (int)w[3]);
    }
}

int launch_requant_staged16(const int16_t* in, const uint8_t* tshift, int64_t rows, int32_t cols,
                            const StageMap& sm, const int32_t* exp_a, const int32_t* exp_b, int bits,
                            int8_t* out, int32_t* out_exp, const unsigned long long* maxp, hipStream_t s,
                            const uint64_t* part, int64_t nparts)
{
    RqArgs a;
    a.part = part; a.nparts = nparts;
    a.n = rows * cols; a.exp_a = exp_a; a.exp_b = exp_b; a.exp_add = 0;
    a.bits = bits; a.stochastic = 0; a.keep_scale = 1;
    a.seed = 0; a.tensor_id = 0; a.step = 0;
    a.out_exp = out_exp; a.maxp = maxp;
    if (cols % 16 || sm.tile_cols % 16 || (((uintptr_t)in | (uintptr_t)out) & 15)) return ISEG_ERR_ARG;
    ISEG_TIMED_LAUNCH(ISEG_KID_REQUANT, s, k_requant_s16_i8, dim3(grid_for(rows * cols, 256 * 16, part ? 1024 : 8192)),
                      dim3(256),
                      0, s, in, tshift, rows, cols, sm, out, a);
    return launch_ok();
}

// ---------------------------------------------------------------------------
// iseg_requant
// ---------------------------------------------------------------------------
extern "C" size_t iseg_requant_ws(int64_t) { return 256; }

extern "C" int iseg_requant(const void* in, int32_t in_dtype, int64_t n, const int32_t* in_exp,
                            int32_t bits, int32_t stochastic, int32_t keep_scale,
                            uint64_t seed, uint32_t tensor_id, uint32_t step,
                            int32_t out_dtype, void* out, int32_t* out_exp,
                            void* ws, size_t ws_bytes, int32_t* dev_status, hipStream_t stream)
{
    if (n < 0 || !out_exp || (n > 0 && (!in || !out))) return ISEG_ERR_ARG;
    if (in_dtype != ISEG_I32 && in_dtype != ISEG_I64) return ISEG_ERR_ARG;
    if (out_dtype == ISEG_I8 ? (bits < 2 || bits > 8)
                             : (out_dtype != ISEG_I16 || bits < 2 || bits > 16))
        return ISEG_ERR_ARG;
    if (keep_scale && !in_exp) return ISEG_ERR_ARG;
    if (!ws || ws_bytes < iseg_requant_ws(n)) return ISEG_ERR_WORKSPACE;
    unsigned long long* maxp = (unsigned long long*)ws;
    int rc = launch_fill_u32(maxp, 2, 0, stream);
    if (rc == ISEG_OK) rc = launch_absmax(in, in_dtype, n, maxp, dev_status, stream);
    if (rc == ISEG_OK)
        rc = launch_requant_apply(in, in_dtype, n, keep_scale ? in_exp : nullptr, nullptr, 0,
                                  bits, stochastic, keep_scale, seed, tensor_id, step,
                                  out_dtype, out, out_exp, maxp, stream);
    return rc;
}

// ---------------------------------------------------------------------------
// iseg_quantize: float32 -> codes
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_fabsmax(const float* __restrict__ x, int64_t n,
                                                 unsigned long long* maxp, int32_t* dev_status)
{
    uint32_t m = 0;
    bool bad = false;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        uint32_t b = __float_as_uint(x[i]) & 0x7fffffffu;
        bad |= b >= 0x7f800000u;
        m = b > m ? b : m;
    }
    if (bad) set_status(dev_status, ISEG_DEV_NONFINITE);
    block_atomic_max_u64(m, maxp);
}

// exponent e of the smallest power of two strictly greater than the positive
// float with bits `mb` (frexp's exponent)
__device__ __forceinline__ int frexp_exp_bits(uint32_t mb)
{
    uint32_t E = mb >> 23, man = mb & 0x7fffffu;
    if (E == 0) return bitlen_u64(man) - 149;
    return (int)E - 126;
}

struct QzArgs {
    int64_t n;
    int32_t bits, mode;
    int32_t* out_exp;
    const unsigned long long* maxp;
};

template <typename TOut>
__global__ __launch_bounds__(256) void k_quantize_apply(const float* __restrict__ x,
                                                        TOut* __restrict__ out, QzArgs a)
{
    int b = 0;
    if (a.mode == ISEG_Q_SQ) {
        uint32_t mb = (uint32_t)*a.maxp;
        b = mb ? frexp_exp_bits(mb) : 0;
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) *a.out_exp = b + 1 - a.bits;
    int sh = a.bits - 1 - b;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < a.n;
         i += (int64_t)gridDim.x * blockDim.x) {
        float v = ldexpf(x[i], sh);         // x / (S Delta), a power-of-two scale
        float fl = floorf(v);
        float fr = v - fl;                  // decides the half-up rounding exactly
        float nf = fl + (fr >= 0.5f ? 1.0f : 0.0f);
        int64_t n;
        if (!(nf == nf)) n = 0;
        else if (nf >= 4.6e18f) n = INT64_MAX / 2;
        else if (nf <= -4.6e18f) n = -(INT64_MAX / 2);
        else n = (int64_t)nf;
        out[i] = (TOut)clamp_k(n, a.bits);
    }
}

extern "C" size_t iseg_quantize_ws(int64_t) { return 256; }

extern "C" int iseg_quantize(const float* x, int64_t n, int32_t bits, int32_t mode,
                             int32_t out_dtype, void* out, int32_t* out_exp,
                             void* ws, size_t ws_bytes, int32_t* dev_status, hipStream_t stream)
{
    if (n < 0 || !out_exp || (n > 0 && (!x || !out))) return ISEG_ERR_ARG;
    if (mode != ISEG_Q_UQ && mode != ISEG_Q_SQ) return ISEG_ERR_ARG;
    int maxbits = out_dtype == ISEG_I8 ? 8 : out_dtype == ISEG_I16 ? 16 : out_dtype == ISEG_I32 ? 31 : 0;
    if (bits < 2 || bits > maxbits) return ISEG_ERR_ARG;
    if (!ws || ws_bytes < iseg_quantize_ws(n)) return ISEG_ERR_WORKSPACE;
    unsigned long long* maxp = (unsigned long long*)ws;
    int rc = launch_fill_u32(maxp, 2, 0, stream);
    if (rc != ISEG_OK) return rc;
    if (n > 0) {
        hipLaunchKernelGGL(k_fabsmax, dim3(grid_for(n, 256 * 8, 2048)), dim3(256), 0, stream,
                           x, n, maxp, dev_status);
        if ((rc = launch_ok()) != ISEG_OK) return rc;
    }
    QzArgs a;
    a.n = n; a.bits = bits; a.mode = mode; a.out_exp = out_exp; a.maxp = maxp;
    dim3 g(grid_for(n, 256 * 4, 4096));
    if (out_dtype == ISEG_I8)
        hipLaunchKernelGGL(k_quantize_apply<int8_t>, g, dim3(256), 0, stream, x, (int8_t*)out, a);
    else if (out_dtype == ISEG_I16)
        hipLaunchKernelGGL(k_quantize_apply<int16_t>, g, dim3(256), 0, stream, x, (int16_t*)out, a);
    else
        hipLaunchKernelGGL(k_quantize_apply<int32_t>, g, dim3(256), 0, stream, x, (int32_t*)out, a);
    return launch_ok();
}

// ---------------------------------------------------------------------------
// Eq. 19 update and Eq. 8 weight quantizer
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_weight_update(int32_t* __restrict__ master, int64_t n,
                                                       const int8_t* __restrict__ g,
                                                       const int32_t* g_exp, int32_t lr_shift,
                                                       int32_t master_exp, int32_t k_U,
                                                       int32_t k_W, int8_t* __restrict__ w_q)
{
    int sh = *g_exp - lr_shift - master_exp;     // Delta W code = g 2^sh, rounded
    int dq = k_U - k_W;
    int64_t lim = ((int64_t)1 << (k_U - 1)) - 1;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        int64_t gv = g[i];
        int64_t dW;
        if (gv == 0 || sh < -40) dW = 0;
        else if (sh > 40) dW = gv > 0 ? lim : -lim;
        else if (sh >= 0) dW = clamp_k(gv * ((int64_t)1 << sh), k_U);
        else dW = clamp_k(shr_rhu(gv, -sh), k_U);
        int64_t m = clamp_k((int64_t)master[i] - dW, k_U);
        master[i] = (int32_t)m;
        w_q[i] = (int8_t)clamp_k(shr_rhu(m, dq), k_W);
    }
}

extern "C" int iseg_weight_update(int32_t* master, int64_t n, const int8_t* g, const int32_t* g_exp,
                                  int32_t lr_shift, int32_t master_exp, int32_t k_U, int32_t k_W,
                                  int8_t* w_q, int32_t*, hipStream_t stream)
{
    if (n < 0 || (n > 0 && (!master || !g || !g_exp || !w_q))) return ISEG_ERR_ARG;
    if (k_U < 9 || k_U > 31 || k_W < 2 || k_W > 8) return ISEG_ERR_ARG;
    if (n == 0) return ISEG_OK;
    hipLaunchKernelGGL(k_weight_update, dim3(grid_for(n, 256, 4096)), dim3(256), 0, stream,
                       master, n, g, g_exp, lr_shift, master_exp, k_U, k_W, w_q);
    return launch_ok();
}

// Q_G + Q_U of gamma (block 0) and beta (block 1) of one L1BN layer
struct BnpArgs {
    const int64_t* d[2];
    const int32_t* dexp[2];
    int32_t* master[2];
    int8_t* wq[2];
    int8_t* gout[2];
    int32_t* gexp[2];
    uint32_t tid[2];
    int64_t C;
    uint64_t seed;
    uint32_t step;
    int32_t bits, lr_shift, master_exp, k_U, k_W;
};

__global__ __launch_bounds__(256) void k_bn_param_update(BnpArgs a)
{
    __shared__ uint64_t red[4];
    const int which = blockIdx.x;
    const int64_t* d = a.d[which];
    uint64_t m = 0;
    for (int64_t c = threadIdx.x; c < a.C; c += blockDim.x) {
        uint64_t v = uabs64(d[c]);
        m = v > m ? v : m;
    }
    m = wave_max_u64(m);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
    __syncthreads();
    m = red[0];
    for (int i = 1; i < 4; i++) m = red[i] > m ? red[i] : m;
    const int r = m ? bitlen_u64(m) - (a.bits - 1) : 0;
    const int32_t gexp = *a.dexp[which] + r;                   // Eq. 17 keeps the scale
    if (threadIdx.x == 0 && a.gexp[which]) *a.gexp[which] = gexp;
    const int sh = gexp - a.lr_shift - a.master_exp;
    const int dq = a.k_U - a.k_W;
    const int64_t lim = ((int64_t)1 << (a.k_U - 1)) - 1;
    for (int64_t c = threadIdx.x; c < a.C; c += blockDim.x) {
        int64_t g = r > 0 ? rq_code(d[c], r, a.bits, philox_draw(a.seed, a.tid[which], a.step, (uint64_t)c))
                          : sq_code(d[c], r, a.bits);
        if (a.gout[which]) a.gout[which][c] = (int8_t)g;
        int64_t dW;
        if (g == 0 || sh < -40) dW = 0;
        else if (sh > 40) dW = g > 0 ? lim : -lim;
        else if (sh >= 0) dW = clamp_k(g * ((int64_t)1 << sh), a.k_U);
        else dW = clamp_k(shr_rhu(g, -sh), a.k_U);
        int64_t mm = clamp_k((int64_t)a.master[which][c] - dW, a.k_U);
        a.master[which][c] = (int32_t)mm;
        a.wq[which][c] = (int8_t)clamp_k(shr_rhu(mm, dq), a.k_W);
    }
}

extern "C" int iseg_bn_param_update(const int64_t* dgamma, const int32_t* dgamma_exp,
                                    const int64_t* dbeta, const int32_t* dbeta_exp, int64_t C,
                                    int32_t bits, uint64_t seed, uint32_t tid_gamma, uint32_t tid_beta,
                                    uint32_t step, int32_t lr_shift, int32_t master_exp, int32_t k_U,
                                    int32_t k_W, int32_t* gamma_m, int32_t* beta_m, int8_t* gamma_q,
                                    int8_t* beta_q, int8_t* g_gamma, int8_t* g_beta,
                                    int32_t* g_gamma_exp, int32_t* g_beta_exp, int32_t*,
                                    hipStream_t stream)
{
    if (C < 1 || !dgamma || !dgamma_exp || !dbeta || !dbeta_exp || !gamma_m || !beta_m ||
        !gamma_q || !beta_q)
        return ISEG_ERR_ARG;
    if (bits < 2 || bits > 8 || k_U < 9 || k_U > 31 || k_W < 2 || k_W > 8) return ISEG_ERR_ARG;
    BnpArgs a;
    a.d[0] = dgamma; a.d[1] = dbeta;
    a.dexp[0] = dgamma_exp; a.dexp[1] = dbeta_exp;
    a.master[0] = gamma_m; a.master[1] = beta_m;
    a.wq[0] = gamma_q; a.wq[1] = beta_q;
    a.gout[0] = g_gamma; a.gout[1] = g_beta;
    a.gexp[0] = g_gamma_exp; a.gexp[1] = g_beta_exp;
    a.tid[0] = tid_gamma; a.tid[1] = tid_beta;
    a.C = C; a.seed = seed; a.step = step;
    a.bits = bits; a.lr_shift = lr_shift; a.master_exp = master_exp; a.k_U = k_U; a.k_W = k_W;
    hipLaunchKernelGGL(k_bn_param_update, dim3(2), dim3(256), 0, stream, a);
    return launch_ok();
}

// ---------------------------------------------------------------------------
// every parameter of a network in one launch: block (x, t) takes part of
// descriptor t.  ISEG_UPD_CODES tensors (conv weights, G already quantized by
// Q_G) are split over the x blocks; ISEG_UPD_RAW tensors (L1BN gamma / beta:
// raw int64 sums, Q_G = stochastic RQ with the tensor's max first) are small
// and handled by block x = 0 alone.
// ---------------------------------------------------------------------------
struct UpdCfg {
    uint64_t seed;
    uint32_t step;
    int32_t bits, lr_shift, k_U, k_W;
};

__device__ __forceinline__ int64_t upd_delta(int64_t g, int sh, int k_U, int64_t lim)
{
    if (g == 0 || sh < -40) return 0;
    if (sh > 40) return g > 0 ? lim : -lim;
    if (sh >= 0) return clamp_k(g * ((int64_t)1 << sh), k_U);
    return clamp_k(shr_rhu(g, -sh), k_U);
}

// Work split into chunks of kUpdChunk elements over all ISEG_UPD_CODES
// tensors (one chunk per ISEG_UPD_RAW tensor, which one block handles whole);
// a fixed grid strides over the chunks, each block first forming the chunk
// offsets of the descriptors in LDS.
constexpr int kUpdChunk = 4096;
constexpr int kUpdMaxDesc = 4096;

__global__ __launch_bounds__(256) void k_update_multi(const iseg_update_desc* __restrict__ descs, int n_desc,
                                                      UpdCfg u, int32_t* __restrict__ dev_status)
{
    __shared__ int32_t first[kUpdMaxDesc + 1];
    __shared__ int32_t tot[256];
    __shared__ uint64_t red[4];
    {
        // chunk counts of a run of descriptors per thread (loads in parallel),
        // then an exclusive scan of the per-thread totals
        const int per = (n_desc + 255) / 256;
        const int d0 = threadIdx.x * per;
        int32_t t = 0;
        for (int d = d0; d < d0 + per && d < n_desc; d++) {
            const int32_t c = descs[d].kind == ISEG_UPD_CODES ? (int32_t)((descs[d].n + kUpdChunk - 1) / kUpdChunk) : 1;
            first[d] = c;
            t += c;
        }
        tot[threadIdx.x] = t;
        __syncthreads();
        if (threadIdx.x == 0) {
            int32_t acc = 0;
            for (int i = 0; i < 256; i++) {
                const int32_t v = tot[i];
                tot[i] = acc;
                acc += v;
            }
            first[n_desc] = acc;
        }
        __syncthreads();
        int32_t acc = tot[threadIdx.x];
        for (int d = d0; d < d0 + per && d < n_desc; d++) {
            const int32_t c = first[d];
            first[d] = acc;
            acc += c;
        }
        __syncthreads();
    }
    const int nchunks = first[n_desc];
    const int64_t lim = ((int64_t)1 << (u.k_U - 1)) - 1;
    for (int ch = blockIdx.x; ch < nchunks; ch += gridDim.x) {
        int lo = 0, hi = n_desc - 1;                 // last descriptor with first <= ch
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (first[mid] <= ch) lo = mid;
            else hi = mid - 1;
        }
        const iseg_update_desc d = descs[lo];
        const int kw = d.k_w ? d.k_w : u.k_W;                        // Q_W width of this tensor
        if (kw < 2 || kw > 8) {
            if (threadIdx.x == 0) set_status(dev_status, ISEG_DEV_DESC);
            continue;
        }
        const int dq = u.k_U - kw;
        if (d.kind == ISEG_UPD_CODES) {
            const int8_t* g = (const int8_t*)d.g;
            const int sh = *d.g_exp - u.lr_shift - d.master_exp;      // Delta W code = g 2^sh, rounded
            const int64_t i0 = (int64_t)(ch - first[lo]) * kUpdChunk;
            const int64_t i1 = i0 + kUpdChunk < d.n ? i0 + kUpdChunk : d.n;
            // four elements per thread step when the tensors allow 16-byte
            // master and 4-byte code accesses (chunk starts are multiples of 4)
            const bool vec = ((((uintptr_t)d.master) & 15) | (((uintptr_t)g) & 3) | (((uintptr_t)d.w_q) & 3)) == 0;
            const int64_t n4 = vec ? (i1 - i0) >> 2 : 0;
            for (int64_t q = threadIdx.x; q < n4; q += blockDim.x) {
                const int64_t i = i0 + 4 * q;
                const int4 mv = *(const int4*)(d.master + i);
                const uint32_t gv = *(const uint32_t*)(g + i);
                int32_t mm[4] = {mv.x, mv.y, mv.z, mv.w};
                uint32_t wq = 0;
#pragma unroll
                for (int e = 0; e < 4; e++) {
                    const int64_t m =
                        clamp_k((int64_t)mm[e] - upd_delta((int8_t)(gv >> (8 * e)), sh, u.k_U, lim), u.k_U);
                    mm[e] = (int32_t)m;
                    wq |= (uint32_t)(uint8_t)(int8_t)clamp_k(shr_rhu(m, dq), kw) << (8 * e);
                }
                *(int4*)(d.master + i) = make_int4(mm[0], mm[1], mm[2], mm[3]);
                *(uint32_t*)(d.w_q + i) = wq;
            }
            for (int64_t i = i0 + 4 * n4 + threadIdx.x; i < i1; i += blockDim.x) {
                const int64_t m = clamp_k((int64_t)d.master[i] - upd_delta(g[i], sh, u.k_U, lim), u.k_U);
                d.master[i] = (int32_t)m;
                d.w_q[i] = (int8_t)clamp_k(shr_rhu(m, dq), kw);
            }
            continue;
        }
        const int64_t* g = (const int64_t*)d.g;
        uint64_t m = 0;
        for (int64_t c = threadIdx.x; c < d.n; c += blockDim.x) {
            const uint64_t v = uabs64(g[c]);
            m = v > m ? v : m;
        }
        m = wave_max_u64(m);
        if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
        __syncthreads();
        m = red[0];
        for (int i = 1; i < (int)(blockDim.x >> 6); i++) m = red[i] > m ? red[i] : m;
        __syncthreads();
        const int r = m ? bitlen_u64(m) - (u.bits - 1) : 0;
        const int32_t gexp = *d.g_exp + r;                             // Eq. 17 keeps the scale
        if (threadIdx.x == 0 && d.g_q_exp) *d.g_q_exp = gexp;
        const int sh = gexp - u.lr_shift - d.master_exp;
        for (int64_t c = threadIdx.x; c < d.n; c += blockDim.x) {
            const int64_t q = r > 0 ? rq_code(g[c], r, u.bits, philox_draw(u.seed, d.tensor_id, u.step, (uint64_t)c))
                                    : sq_code(g[c], r, u.bits);
            if (d.g_q) d.g_q[c] = (int8_t)q;
            const int64_t mm = clamp_k((int64_t)d.master[c] - upd_delta(q, sh, u.k_U, lim), u.k_U);
            d.master[c] = (int32_t)mm;
            d.w_q[c] = (int8_t)clamp_k(shr_rhu(mm, dq), kw);
        }
    }
}

extern "C" int iseg_update_multi(const iseg_update_desc* descs, int32_t n_desc, int32_t bits, uint64_t seed,
                                 uint32_t step, int32_t lr_shift, int32_t k_U, int32_t k_W, int32_t* dev_status,
                                 hipStream_t stream)
{
    if (n_desc < 0 || n_desc > kUpdMaxDesc || (n_desc > 0 && !descs)) return ISEG_ERR_ARG;
    if (bits < 2 || bits > 8 || k_U < 9 || k_U > 31 || k_W < 2 || k_W > 8) return ISEG_ERR_ARG;
    if (n_desc == 0) return ISEG_OK;
    UpdCfg u;
    u.seed = seed; u.step = step; u.bits = bits; u.lr_shift = lr_shift; u.k_U = k_U; u.k_W = k_W;
    hipLaunchKernelGGL(k_update_multi, dim3(2048), dim3(256), 0, stream, descs, (int)n_desc, u,
                       dev_status);
    return launch_ok();
}

__global__ __launch_bounds__(256) void k_weight_quant(const int32_t* __restrict__ master, int64_t n,
                                                      int32_t dq, int32_t k_W, int8_t* __restrict__ w_q)
{
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        w_q[i] = (int8_t)clamp_k(shr_rhu(master[i], dq), k_W);
}

extern "C" int iseg_weight_quant(const int32_t* master, int64_t n, int32_t k_U, int32_t k_W,
                                 int8_t* w_q, hipStream_t stream)
{
    if (n < 0 || (n > 0 && (!master || !w_q))) return ISEG_ERR_ARG;
    if (k_U < 9 || k_U > 31 || k_W < 2 || k_W > 8) return ISEG_ERR_ARG;
    if (n == 0) return ISEG_OK;
    hipLaunchKernelGGL(k_weight_quant, dim3(grid_for(n, 256, 4096)), dim3(256), 0, stream,
                       master, n, k_U - k_W, k_W, w_q);
    return launch_ok();
}

// ---------------------------------------------------------------------------
// host utilities
// ---------------------------------------------------------------------------
extern "C" void iseg_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4])
{
    philox_out o = philox4x32_10(ctr[0], ctr[1], ctr[2], ctr[3], key[0], key[1]);
    for (int i = 0; i < 4; i++) out[i] = o.v[i];
}

extern "C" const char* iseg_version(void) { return "iseg 0.1 gfx950"; }
