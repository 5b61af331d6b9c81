// pool.hip -- max pooling on int8 codes (encoder glue of the VGG16 / ResNet-50
// encoders) and its backward.  The forward picks the first maximum in
// row-major window order (padding is never picked) and keeps the exponent;
// the backward routes each error code to that position, adds overlapping
// windows exactly in int32 and applies Q_E (SQ, Eq. 16) to the sums.
#include "iseg_common.h"

namespace {

struct PoolGeom {
    int64_t N, H, W, C, P, Q;
    int32_t k, st, pad;
};

__device__ __forceinline__ int64_t pool_argmax(const int8_t* __restrict__ x, const PoolGeom& g,
                                               int64_t n, int p, int q, int64_t c)
{
    int64_t best = -1;
    int bv = -1000;
    for (int r = 0; r < g.k; r++) {
        int h = p * g.st - g.pad + r;
        if (h < 0 || h >= g.H) continue;
        for (int s = 0; s < g.k; s++) {
            int w = q * g.st - g.pad + s;
            if (w < 0 || w >= g.W) continue;
            int64_t idx = ((n * g.H + h) * g.W + w) * g.C + c;
            int v = x[idx];
            if (v > bv) { bv = v; best = idx; }
        }
    }
    return best;
}

__global__ __launch_bounds__(256) void k_maxpool_fwd(const int8_t* __restrict__ x, int8_t* __restrict__ y,
                                                     PoolGeom g, const int32_t* x_exp, int32_t* y_exp)
{
    if (blockIdx.x == 0 && threadIdx.x == 0) *y_exp = *x_exp;
    int64_t total = g.N * g.P * g.Q * g.C;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        int64_t c = i % g.C;
        int64_t t = i / g.C;
        int q = (int)(t % g.Q);
        t /= g.Q;
        int p = (int)(t % g.P);
        int64_t n = t / g.P;
        int64_t a = pool_argmax(x, g, n, p, q, c);
        y[i] = a >= 0 ? x[a] : 0;
    }
}

__global__ __launch_bounds__(256) void k_maxpool_bwd(const int8_t* __restrict__ dy,
                                                     const int8_t* __restrict__ x,
                                                     int32_t* __restrict__ acc, PoolGeom g,
                                                     unsigned long long* maxp)
{
    int64_t total = g.N * g.H * g.W * g.C;
    uint64_t mx = 0;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        int64_t c = i % g.C;
        int64_t t = i / g.C;
        int w = (int)(t % g.W);
        t /= g.W;
        int h = (int)(t % g.H);
        int64_t n = t / g.H;
        // windows p with p*st - pad <= h <= p*st - pad + k - 1
        int plo = h + g.pad - g.k + 1;
        plo = plo <= 0 ? 0 : (plo + g.st - 1) / g.st;
        int phi = (h + g.pad) / g.st;
        int qlo = w + g.pad - g.k + 1;
        qlo = qlo <= 0 ? 0 : (qlo + g.st - 1) / g.st;
        int qhi = (w + g.pad) / g.st;
        int32_t sum = 0;
        for (int p = plo; p <= phi && p < g.P; p++)
            for (int q = qlo; q <= qhi && q < g.Q; q++)
                if (pool_argmax(x, g, n, p, q, c) == i)
                    sum += dy[((n * g.P + p) * g.Q + q) * g.C + c];
        acc[i] = sum;
        uint64_t a = sum < 0 ? (uint64_t)(-(int64_t)sum) : (uint64_t)sum;
        mx = a > mx ? a : mx;
    }
    block_atomic_max_u64(mx, maxp);
}

// forward, four channels (one dword) per lane
__global__ __launch_bounds__(256) void k_maxpool_fwd4(const int8_t* __restrict__ x, int8_t* __restrict__ y,
                                                      PoolGeom g, const int32_t* x_exp, int32_t* y_exp)
{
    if (blockIdx.x == 0 && threadIdx.x == 0) *y_exp = *x_exp;
    const int64_t C4 = g.C / 4;
    const int64_t total = g.N * g.P * g.Q * C4;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        int64_t c4 = i % C4;
        int64_t t = i / C4;
        int q = (int)(t % g.Q);
        t /= g.Q;
        int p = (int)(t % g.P);
        int64_t n = t / g.P;
        int best[4] = {-1000, -1000, -1000, -1000};
        for (int r = 0; r < g.k; r++) {
            int h = p * g.st - g.pad + r;
            if (h < 0 || h >= g.H) continue;
            for (int s = 0; s < g.k; s++) {
                int w = q * g.st - g.pad + s;
                if (w < 0 || w >= g.W) continue;
                uint32_t v = *(const uint32_t*)(x + ((n * g.H + h) * g.W + w) * g.C + c4 * 4);
#pragma unroll
                for (int j = 0; j < 4; j++) {
                    int b = (int)(int8_t)(v >> (8 * j));
                    best[j] = b > best[j] ? b : best[j];
                }
            }
        }
        uint32_t o = 0;
#pragma unroll
        for (int j = 0; j < 4; j++) o |= (uint32_t)(uint8_t)best[j] << (8 * j);
        *(uint32_t*)(y + i * 4) = o;
    }
}

__global__ __launch_bounds__(256) void k_absmax_i8x4(const int8_t* __restrict__ p, int64_t n4,
                                                     unsigned long long* maxp)
{
    uint64_t m = 0;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n4;
         i += (int64_t)gridDim.x * blockDim.x) {
        uint32_t v = ((const uint32_t*)p)[i];
#pragma unroll
        for (int j = 0; j < 4; j++) {
            int b = (int)(int8_t)(v >> (8 * j));
            uint64_t a = (uint64_t)(b < 0 ? -b : b);
            m = a > m ? a : m;
        }
    }
    block_atomic_max_u64(m, maxp);
}

// backward for non-overlapping windows (k == stride, no padding), one lane per
// input pixel and four channels: each input receives at most one error, so
// max|routed| = max|dy| and the SQ codes are written directly.
__global__ __launch_bounds__(256) void k_maxpool_bwd_disjoint(const int8_t* __restrict__ dy,
                                                              const int8_t* __restrict__ x,
                                                              int8_t* __restrict__ dx, PoolGeom g,
                                                              const unsigned long long* maxp,
                                                              const int32_t* dy_exp, int32_t* dx_exp,
                                                              int bits)
{
    const uint64_t M = *maxp;
    const int r = M ? bitlen_u64(M) - (bits - 1) : 0;
    if (blockIdx.x == 0 && threadIdx.x == 0) *dx_exp = *dy_exp + r;
    const int64_t C4 = g.C / 4;
    const int64_t total = g.N * g.H * g.W * C4;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        int64_t c4 = i % C4;
        int64_t t = i / C4;
        int w = (int)(t % g.W);
        t /= g.W;
        int h = (int)(t % g.H);
        int64_t n = t / g.H;
        int p = h / g.k, q = w / g.k;
        uint32_t o = 0;
        if (p < g.P && q < g.Q) {
            // first maximum of the window in row-major order, per channel
            int best[4] = {-1000, -1000, -1000, -1000}, bpos[4] = {0, 0, 0, 0};
            for (int rr = 0; rr < g.k; rr++)
                for (int s = 0; s < g.k; s++) {
                    uint32_t v = *(const uint32_t*)(x + ((n * g.H + p * g.k + rr) * g.W + q * g.k + s) * g.C + c4 * 4);
#pragma unroll
                    for (int j = 0; j < 4; j++) {
                        int b = (int)(int8_t)(v >> (8 * j));
                        if (b > best[j]) { best[j] = b; bpos[j] = rr * g.k + s; }
                    }
                }
            uint32_t e = *(const uint32_t*)(dy + ((n * g.P + p) * g.Q + q) * g.C + c4 * 4);
            int me = (h - p * g.k) * g.k + (w - q * g.k);
#pragma unroll
            for (int j = 0; j < 4; j++)
                if (bpos[j] == me)
                    o |= (uint32_t)(uint8_t)sq_code((int8_t)(e >> (8 * j)), r, bits) << (8 * j);
        }
        *(uint32_t*)(dx + i * 4) = o;
    }
}

// max |code| of an int8 tensor: one partial per block (no atomics), 16 bytes per load
__global__ __launch_bounds__(256) void k_absmax_i8_part(const int8_t* __restrict__ p, int64_t n16,
                                                        uint64_t* __restrict__ part)
{
    uint32_t m = 0;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n16; i += (int64_t)gridDim.x * blockDim.x) {
        const uint4 v = ((const uint4*)p)[i];
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int q = 0; q < 4; q++)
#pragma unroll
            for (int j = 0; j < 4; j++) {
                const int b = (int)(int8_t)(w[q] >> (8 * j));
                const uint32_t a = (uint32_t)(b < 0 ? -b : b);
                m = a > m ? a : m;
            }
    }
    block_store_max_u64(m, part);
}

// Backward of non-overlapping k x k windows (stride k, no padding), one lane
// per window and 16 channels: the window's k^2 input vectors are read once,
// the first maximum of each channel (row-major order) receives the channel's
// error code and every other input gets 0.  Each input takes at most one
// error, so max |routed| = max |dy| and the SQ codes are final.  Inputs beyond
// the last full window are zeroed by k_pool_zero_tail.
template <int K>
__global__ __launch_bounds__(256) void k_maxpool_bwd_win(const int8_t* __restrict__ dy,
                                                         const int8_t* __restrict__ x, int8_t* __restrict__ dx,
                                                         PoolGeom g, const uint64_t* __restrict__ part, int npart,
                                                         const int32_t* dy_exp, int32_t* dx_exp, int bits)
{
    const uint64_t M = reduce_partials_u64(part, npart);
    const int r = M ? bitlen_u64(M) - (bits - 1) : 0;
    if (blockIdx.x == 0 && threadIdx.x == 0) *dx_exp = *dy_exp + r;
    const int64_t C16 = g.C / 16;
    const int64_t total = g.N * g.P * g.Q * C16;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t cg = i % C16, wi = i / C16;
        const int q = (int)(wi % g.Q);
        const int64_t t = wi / g.Q;
        const int p = (int)(t % g.P);
        const int64_t n = t / g.P;
        uint32_t v[K * K][4];
#pragma unroll
        for (int rr = 0; rr < K; rr++)
#pragma unroll
            for (int s2 = 0; s2 < K; s2++) {
                const uint4 u = *(const uint4*)(x + ((n * g.H + p * K + rr) * g.W + q * K + s2) * g.C + cg * 16);
                v[rr * K + s2][0] = u.x; v[rr * K + s2][1] = u.y; v[rr * K + s2][2] = u.z; v[rr * K + s2][3] = u.w;
            }
        const uint4 eu = *(const uint4*)(dy + ((n * g.P + p) * g.Q + q) * g.C + cg * 16);
        const uint32_t ew[4] = {eu.x, eu.y, eu.z, eu.w};
        uint32_t o[K * K][4];
#pragma unroll
        for (int w = 0; w < K * K; w++)
#pragma unroll
            for (int d = 0; d < 4; d++) o[w][d] = 0;
#pragma unroll
        for (int d = 0; d < 4; d++)
#pragma unroll
            for (int j = 0; j < 4; j++) {
                int best = (int)(int8_t)(v[0][d] >> (8 * j)), bpos = 0;
#pragma unroll
                for (int w = 1; w < K * K; w++) {
                    const int b = (int)(int8_t)(v[w][d] >> (8 * j));
                    if (b > best) { best = b; bpos = w; }
                }
                const uint32_t code = (uint32_t)(uint8_t)sq_code((int8_t)(ew[d] >> (8 * j)), r, bits);
#pragma unroll
                for (int w = 0; w < K * K; w++) o[w][d] |= (bpos == w ? code : 0u) << (8 * j);
            }
#pragma unroll
        for (int rr = 0; rr < K; rr++)
#pragma unroll
            for (int s2 = 0; s2 < K; s2++) {
                const uint32_t* ow = o[rr * K + s2];
                *(uint4*)(dx + ((n * g.H + p * K + rr) * g.W + q * K + s2) * g.C + cg * 16) =
                    make_uint4(ow[0], ow[1], ow[2], ow[3]);
            }
    }
}

// zero the input rows / columns that no full window covers
__global__ __launch_bounds__(256) void k_pool_zero_tail(int8_t* __restrict__ dx, PoolGeom g)
{
    const int64_t C16 = g.C / 16;
    const int64_t total = g.N * g.H * g.W * C16;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t pix = i / C16;
        const int w = (int)(pix % g.W);
        const int h = (int)((pix / g.W) % g.H);
        if (h >= g.P * g.k || w >= g.Q * g.k) *(uint4*)(dx + i * 16) = make_uint4(0, 0, 0, 0);
    }
}

bool pool_geom(int64_t N, int64_t H, int64_t W, int64_t C, int32_t k, int32_t st, int32_t pad,
               PoolGeom* g)
{
    if (N < 0 || H < 1 || W < 1 || C < 1 || k < 1 || st < 1 || pad < 0 || pad >= k) return false;
    if (H + 2 * pad < k || W + 2 * pad < k) return false;
    g->N = N; g->H = H; g->W = W; g->C = C; g->k = k; g->st = st; g->pad = pad;
    g->P = (H + 2 * pad - k) / st + 1;
    g->Q = (W + 2 * pad - k) / st + 1;
    return true;
}

// ---------------------------------------------------------------------------
// Backward for any window / stride / padding, 16 channels per lane:
//   k_pool_argtap16   per output window: the tap (r k + s, row-major) of each
//                     channel's first maximum, one byte per element
//   k_pool_gather16   per input position: the sum of dy over the covering
//                     windows whose tap is this position (at most
//                     ceil(k/st)^2 windows); pass 0 writes per-block max |sum|
//                     partials, pass 1 reduces them and writes the SQ codes
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_pool_argtap16(const int8_t* __restrict__ x, uint8_t* __restrict__ tap,
                                                       PoolGeom g)
{
    const int64_t C16 = g.C / 16;
    const int64_t total = g.N * g.P * g.Q * C16;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t c16 = i % C16;
        int64_t t = i / C16;
        const int q = (int)(t % g.Q);
        t /= g.Q;
        const int p = (int)(t % g.P);
        const int64_t n = t / g.P;
        int best[16], bt[16];
#pragma unroll
        for (int j = 0; j < 16; j++) { best[j] = -1000; bt[j] = 0; }
        for (int r = 0; r < g.k; r++) {
            const int h = p * g.st - g.pad + r;
            if (h < 0 || h >= g.H) continue;
            for (int s2 = 0; s2 < g.k; s2++) {
                const int w = q * g.st - g.pad + s2;
                if (w < 0 || w >= g.W) continue;
                const uint4 v = *(const uint4*)(x + ((n * g.H + h) * g.W + w) * g.C + c16 * 16);
                const uint32_t vw[4] = {v.x, v.y, v.z, v.w};
                const int tp = r * g.k + s2;
#pragma unroll
                for (int j = 0; j < 16; j++) {
                    const int b = (int)(int8_t)(vw[j >> 2] >> (8 * (j & 3)));
                    if (b > best[j]) { best[j] = b; bt[j] = tp; }
                }
            }
        }
        uint32_t o[4] = {0, 0, 0, 0};
#pragma unroll
        for (int j = 0; j < 16; j++) o[j >> 2] |= (uint32_t)(uint8_t)bt[j] << (8 * (j & 3));
        *(uint4*)(tap + i * 16) = make_uint4(o[0], o[1], o[2], o[3]);
    }
}

template <int PASS>
__global__ __launch_bounds__(256) void k_pool_gather16(const int8_t* __restrict__ dy, const uint8_t* __restrict__ tap,
                                                       PoolGeom g, uint64_t* part, int64_t nparts,
                                                       const int32_t* dy_exp, int32_t* dx_exp, int bits,
                                                       int8_t* __restrict__ dx)
{
    int r = 0;
    if (PASS == 1) {
        const uint64_t M = reduce_partials_u64(part, nparts);
        r = M ? bitlen_u64(M) - (bits - 1) : 0;
        if (blockIdx.x == 0 && threadIdx.x == 0) *dx_exp = *dy_exp + r;
    }
    const int64_t C16 = g.C / 16;
    const int64_t total = g.N * g.H * g.W * C16;
    uint64_t mx = 0;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t c16 = i % C16;
        int64_t t = i / C16;
        const int w = (int)(t % g.W);
        t /= g.W;
        const int h = (int)(t % g.H);
        const int64_t n = t / g.H;
        // windows p with p st - pad <= h <= p st - pad + k - 1
        int plo = h + g.pad - g.k + 1;
        plo = plo <= 0 ? 0 : (plo + g.st - 1) / g.st;
        int phi = (h + g.pad) / g.st;
        phi = phi < g.P - 1 ? phi : (int)g.P - 1;
        int qlo = w + g.pad - g.k + 1;
        qlo = qlo <= 0 ? 0 : (qlo + g.st - 1) / g.st;
        int qhi = (w + g.pad) / g.st;
        qhi = qhi < g.Q - 1 ? qhi : (int)g.Q - 1;
        int sum[16];
#pragma unroll
        for (int j = 0; j < 16; j++) sum[j] = 0;
        for (int p = plo; p <= phi; p++)
            for (int q = qlo; q <= qhi; q++) {
                const int me = (h - (p * g.st - g.pad)) * g.k + (w - (q * g.st - g.pad));
                const int64_t o = ((n * g.P + p) * g.Q + q) * g.C + c16 * 16;
                const uint4 tv = *(const uint4*)(tap + o);
                const uint4 dv = *(const uint4*)(dy + o);
                const uint32_t tw[4] = {tv.x, tv.y, tv.z, tv.w}, dw[4] = {dv.x, dv.y, dv.z, dv.w};
#pragma unroll
                for (int j = 0; j < 16; j++)
                    if ((int)((tw[j >> 2] >> (8 * (j & 3))) & 0xff) == me)
                        sum[j] += (int)(int8_t)(dw[j >> 2] >> (8 * (j & 3)));
            }
        if (PASS == 0) {
#pragma unroll
            for (int j = 0; j < 16; j++) {
                const uint64_t a = (uint64_t)(sum[j] < 0 ? -sum[j] : sum[j]);
                mx = a > mx ? a : mx;
            }
        } else {
            uint32_t o[4] = {0, 0, 0, 0};
#pragma unroll
            for (int j = 0; j < 16; j++) o[j >> 2] |= (uint32_t)(uint8_t)sq_code(sum[j], r, bits) << (8 * (j & 3));
            *(uint4*)(dx + i * 16) = make_uint4(o[0], o[1], o[2], o[3]);
        }
    }
    if (PASS == 0) block_store_max_u64(mx, part);
}

}  // namespace

extern "C" int iseg_maxpool_fwd(const int8_t* x, const int32_t* x_exp, int64_t N, int64_t H, int64_t W,
                                int64_t C, int32_t k, int32_t stride, int32_t pad,
                                int8_t* y, int32_t* y_exp, hipStream_t stream)
{
    PoolGeom g;
    if (!pool_geom(N, H, W, C, k, stride, pad, &g)) return ISEG_ERR_SHAPE;
    if (!x_exp || !y_exp || (N > 0 && (!x || !y))) return ISEG_ERR_ARG;
    int64_t total = g.N * g.P * g.Q * g.C;
    if (C % 4 == 0 && (((uintptr_t)x | (uintptr_t)y) & 3) == 0)
        hipLaunchKernelGGL(k_maxpool_fwd4, dim3(grid_for(total / 4, 256, 8192)), dim3(256), 0, stream,
                           x, y, g, x_exp, y_exp);
    else
        hipLaunchKernelGGL(k_maxpool_fwd, dim3(grid_for(total, 256, 8192)), dim3(256), 0, stream,
                           x, y, g, x_exp, y_exp);
    return launch_ok();
}

extern "C" size_t iseg_maxpool_bwd_ws(int64_t N, int64_t H, int64_t W, int64_t C)
{
    return 256 + align256((size_t)(N * H * W * C) * 4);
}

extern "C" int iseg_maxpool_bwd(const int8_t* dy, const int32_t* dy_exp, const int8_t* x,
                                int64_t N, int64_t H, int64_t W, int64_t C,
                                int32_t k, int32_t stride, int32_t pad, int32_t bits,
                                int8_t* dx, int32_t* dx_exp,
                                void* ws, size_t ws_bytes, int32_t* dev_status, hipStream_t stream)
{
    PoolGeom g;
    if (!pool_geom(N, H, W, C, k, stride, pad, &g)) return ISEG_ERR_SHAPE;
    if (!dy_exp || !dx_exp || bits < 2 || bits > 8 || (N > 0 && (!dy || !x || !dx)))
        return ISEG_ERR_ARG;
    if (!ws || ws_bytes < iseg_maxpool_bwd_ws(N, H, W, C)) return ISEG_ERR_WORKSPACE;
    unsigned long long* maxp = (unsigned long long*)ws;
    int32_t* acc = (int32_t*)((char*)ws + 256);
    int rc;
    int64_t total = N * H * W * C;
    if (k == stride && pad == 0 && k == 2 && C % 16 == 0 &&
        (((uintptr_t)x | (uintptr_t)dy | (uintptr_t)dx) & 15) == 0) {
        // per-window routing; the max of dy comes from per-block partials
        uint64_t* part = (uint64_t*)acc;
        const int64_t ndy = g.N * g.P * g.Q * C;
        const unsigned nb = (unsigned)grid_for(ndy / 16, 256 * 4, 256);
        hipLaunchKernelGGL(k_absmax_i8_part, dim3(nb), dim3(256), 0, stream, dy, ndy / 16, part);
        if ((rc = launch_ok())) return rc;
        const int64_t nwin = g.N * g.P * g.Q * (C / 16);
        ISEG_TIMED_LAUNCH(ISEG_KID_MAXPOOL_BWD, stream, k_maxpool_bwd_win<2>, dim3(grid_for(nwin, 256, 8192)),
                          dim3(256), 0, stream, dy, x, dx, g, part, (int)nb, dy_exp, dx_exp, bits);
        if ((rc = launch_ok())) return rc;
        if (g.P * k < H || g.Q * k < W) {
            hipLaunchKernelGGL(k_pool_zero_tail, dim3(grid_for(total / 16, 256, 4096)), dim3(256), 0, stream, dx, g);
            if ((rc = launch_ok())) return rc;
        }
        return ISEG_OK;
    }
    const size_t tap_need = align256((size_t)(g.N * g.P * g.Q * C)) + 1024 * 8;
    if (C % 16 == 0 && k <= 15 && (((uintptr_t)x | (uintptr_t)dy | (uintptr_t)dx) & 15) == 0 && total > 0 &&
        tap_need <= align256((size_t)total * 4)) {
        // any window: per-window argmax taps, then two gathers (max, codes)
        uint8_t* tap = (uint8_t*)acc;
        uint64_t* part = (uint64_t*)((char*)acc + align256((size_t)(g.N * g.P * g.Q * C)));
        const int64_t nwin = g.N * g.P * g.Q * (C / 16);
        hipLaunchKernelGGL(k_pool_argtap16, dim3(grid_for(nwin, 256, 8192)), dim3(256), 0, stream, x, tap, g);
        if ((rc = launch_ok())) return rc;
        const unsigned nb = grid_for(total / 16, 256, 1024);
        ISEG_TIMED_LAUNCH(ISEG_KID_MAXPOOL_BWD, stream, k_pool_gather16<0>, dim3(nb), dim3(256), 0, stream, dy, tap,
                          g, part, (int64_t)nb, dy_exp, dx_exp, bits, dx);
        if ((rc = launch_ok())) return rc;
        hipLaunchKernelGGL(k_pool_gather16<1>, dim3(grid_for(total / 16, 256, 4096)), dim3(256), 0, stream, dy, tap,
                           g, part, (int64_t)nb, dy_exp, dx_exp, bits, dx);
        return launch_ok();
    }
    if ((rc = launch_fill_u32(maxp, 2, 0, stream))) return rc;
    if (k == stride && pad == 0 && C % 4 == 0 &&
        (((uintptr_t)x | (uintptr_t)dy | (uintptr_t)dx) & 3) == 0) {
        int64_t ndy = g.N * g.P * g.Q * C;
        if (ndy > 0)
            hipLaunchKernelGGL(k_absmax_i8x4, dim3(grid_for(ndy / 4, 256 * 4, 2048)), dim3(256), 0,
                               stream, dy, ndy / 4, maxp);
        if ((rc = launch_ok())) return rc;
        ISEG_TIMED_LAUNCH(ISEG_KID_MAXPOOL_BWD, stream, k_maxpool_bwd_disjoint,
                          dim3(grid_for(total / 4, 256, 8192)), dim3(256), 0, stream, dy, x, dx, g,
                          maxp, dy_exp, dx_exp, bits);
        return launch_ok();
    }
    if (total > 0) {
        ISEG_TIMED_LAUNCH(ISEG_KID_MAXPOOL_BWD, stream, k_maxpool_bwd, dim3(grid_for(total, 256, 8192)),
                          dim3(256), 0, stream, dy, x, acc, g, maxp);
        if ((rc = launch_ok())) return rc;
    }
    (void)dev_status;
    return launch_requant_apply(acc, ISEG_I32, total, dy_exp, nullptr, 0, bits, 0, 1, 0, 0, 0,
                                ISEG_I8, dx, dx_exp, maxp, stream);
}
