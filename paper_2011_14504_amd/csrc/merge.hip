// merge.hip -- merges of quantized tensors on gfx950.
//
// Every tensor of the dataflow is an 8-bit object with one power-of-two scale
// (Sec. 3.1, Eq. 3-4).  A residual add, the sum of the errors a tensor gets
// back from several consumers, a channel concatenation and a spatial sum
// (global average pooling, the backward of a spatial broadcast) form their
// exact result on the grid 2^min(e_i) in int64 and requantize it once (SQ,
// Eq. 4 / Eq. 16).  All of these are streaming, bandwidth-bound passes:
//   pass 1: exact result -> per-block max |.| partials (no same-address atomics)
//   pass 2: every block reduces the partials, then writes the codes.
#include <limits.h>

#include "iseg_common.h"

namespace {

constexpr int kMaxIn = 8;
constexpr int kMaxGap = 48;        // aligned int8 terms stay below 2^55
constexpr int kMaxPartials = 1024; // pass-1 grid cap (partials reduced by each pass-2 block)
constexpr int kU = 4;              // 16-byte vectors in flight per lane

struct MergeArgs {
    const int8_t* p[kMaxIn];
    const int32_t* e[kMaxIn];
    int32_t add[kMaxIn];
    int32_t bc[kMaxIn];            // 1: [N,1,1,C] input broadcast over HW
    int32_t any_bc;                // some input is broadcast (its element index needs (n, c))
    int32_t n_in;
    int64_t n, HW, C;
    int32_t relu, bits;
    uint64_t* part;
    int8_t* out;
    int32_t* out_exp;
    int32_t* status;
};

// per-input left shifts onto the common grid 2^e0; false if the gap is too large
__device__ __forceinline__ bool merge_shifts(const MergeArgs& a, int* sh, int* e0_out)
{
    int e[kMaxIn];
    int lo = INT_MAX, hi = INT_MIN;
    for (int i = 0; i < a.n_in; i++) {
        e[i] = *a.e[i] + a.add[i];
        lo = e[i] < lo ? e[i] : lo;
        hi = e[i] > hi ? e[i] : hi;
    }
    for (int i = 0; i < a.n_in; i++) {
        const int d = e[i] - lo;
        sh[i] = d > kMaxGap ? kMaxGap : d;
    }
    *e0_out = lo;
    return hi - lo <= kMaxGap;
}

// exact sums of 16 consecutive elements starting at element j (same image,
// 16 consecutive channels): vector loads of every input
__device__ __forceinline__ void merge_sum16(const MergeArgs& a, const int* sh, int64_t j, int64_t* s)
{
#pragma unroll
    for (int t = 0; t < 16; t++) s[t] = 0;
    const int64_t img = j / (a.HW * a.C);
    const int64_t c = j % a.C;
    for (int i = 0; i < a.n_in; i++) {
        const int64_t src = a.bc[i] ? img * a.C + c : j;
        const int4 v = *(const int4*)(a.p[i] + src);
        const int32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int t = 0; t < 16; t++) {
            const int64_t q = (int8_t)(w[t >> 2] >> (8 * (t & 3)));
            s[t] += q << sh[i];
        }
    }
    if (a.relu) {
#pragma unroll
        for (int t = 0; t < 16; t++) s[t] = s[t] > 0 ? s[t] : 0;
    }
}

// the 16-byte vectors of every input for output vector v (v < nv); the
// (image, channel) split of the element index only when an input is broadcast
template <int NIN>
__device__ __forceinline__ void merge_load16(const MergeArgs& a, int64_t v, int64_t nv, int4* raw)
{
    if (v >= nv) return;
    const int64_t j = v * 16;
    if (!a.any_bc) {
#pragma unroll
        for (int i = 0; i < NIN; i++) raw[i] = *(const int4*)(a.p[i] + j);
        return;
    }
    const int64_t img = j / (a.HW * a.C);
    const int64_t c = j % a.C;
#pragma unroll
    for (int i = 0; i < NIN; i++) raw[i] = *(const int4*)(a.p[i] + (a.bc[i] ? img * a.C + c : j));
}

// exact sums of 16 elements on the grid 2^e0 in T: int32 when every shift is
// at most kW32Shift (eight int8 terms stay below 2^31), else int64
constexpr int kW32Shift = 20;
template <int NIN, typename T>
__device__ __forceinline__ void merge_sum16_raw(const MergeArgs& a, const int* sh, const int4* raw, T* s)
{
#pragma unroll
    for (int t = 0; t < 16; t++) s[t] = 0;
#pragma unroll
    for (int i = 0; i < NIN; i++) {
        const int32_t w[4] = {raw[i].x, raw[i].y, raw[i].z, raw[i].w};
#pragma unroll
        for (int t = 0; t < 16; t++) s[t] += (T)(int8_t)(w[t >> 2] >> (8 * (t & 3))) << sh[i];
    }
    if (a.relu) {
#pragma unroll
        for (int t = 0; t < 16; t++) s[t] = s[t] > 0 ? s[t] : 0;
    }
}

// SQ code of an int32 on a given shift (r <= 0 only when max |q| < 2^(k-1))
__device__ __forceinline__ int32_t sq_code32(int32_t q, int r, int k)
{
    const int32_t lim = (1 << (k - 1)) - 1;
    const int32_t v = r > 0 ? (q + (1 << (r - 1))) >> r : q << -r;
    return v > lim ? lim : (v < -lim ? -lim : v);
}

__device__ __forceinline__ int max_shift(const MergeArgs& a, const int* sh)
{
    int m = 0;
    for (int i = 0; i < a.n_in; i++) m = sh[i] > m ? sh[i] : m;
    return m;
}

__device__ __forceinline__ int64_t merge_sum1(const MergeArgs& a, const int* sh, int64_t j)
{
    const int64_t img = j / (a.HW * a.C);
    const int64_t c = j % a.C;
    int64_t s = 0;
    for (int i = 0; i < a.n_in; i++) {
        const int64_t src = a.bc[i] ? img * a.C + c : j;
        s += (int64_t)a.p[i][src] << sh[i];
    }
    if (a.relu && s < 0) s = 0;
    return s;
}

template <bool VEC, int NIN>
__global__ __launch_bounds__(256) void k_merge_max(MergeArgs a)
{
    int sh[kMaxIn], e0;
    if (!merge_shifts(a, sh, &e0) && blockIdx.x == 0 && threadIdx.x == 0) set_status(a.status, ISEG_DEV_RANGE);
    uint64_t m = 0;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t t0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (VEC && NIN > 0) {
        const int64_t nv = a.n / 16;
        const bool w32 = max_shift(a, sh) <= kW32Shift;
        uint32_t m32 = 0;
        for (int64_t v0 = t0; v0 < nv; v0 += stride * kU) {
            int4 raw[kU][NIN > 0 ? NIN : 1];
#pragma unroll
            for (int u = 0; u < kU; u++) merge_load16<NIN>(a, v0 + u * stride, nv, raw[u]);
#pragma unroll
            for (int u = 0; u < kU; u++) {
                if (v0 + u * stride >= nv) break;
                if (w32) {
                    int32_t s[16];
                    merge_sum16_raw<NIN>(a, sh, raw[u], s);
#pragma unroll
                    for (int t = 0; t < 16; t++) m32 = max(m32, (uint32_t)abs(s[t]));
                } else {
                    int64_t s[16];
                    merge_sum16_raw<NIN>(a, sh, raw[u], s);
#pragma unroll
                    for (int t = 0; t < 16; t++) {
                        const uint64_t w = (uint64_t)(s[t] < 0 ? -s[t] : s[t]);
                        m = w > m ? w : m;
                    }
                }
            }
        }
        m = m > m32 ? m : m32;
    } else if (VEC) {
        for (int64_t v = t0; v < a.n / 16; v += stride) {
            int64_t s[16];
            merge_sum16(a, sh, v * 16, s);
#pragma unroll
            for (int t = 0; t < 16; t++) {
                const uint64_t w = (uint64_t)(s[t] < 0 ? -s[t] : s[t]);
                m = w > m ? w : m;
            }
        }
    } else {
        for (int64_t j = t0; j < a.n; j += stride) {
            const int64_t s = merge_sum1(a, sh, j);
            const uint64_t u = (uint64_t)(s < 0 ? -s : s);
            m = u > m ? u : m;
        }
    }
    block_store_max_u64(m, a.part);
}

template <bool VEC, int NIN>
__global__ __launch_bounds__(256) void k_merge_apply(MergeArgs a, int64_t nparts)
{
    int sh[kMaxIn], e0;
    merge_shifts(a, sh, &e0);
    const uint64_t M = reduce_partials_u64(a.part, nparts);
    const int r = M ? bitlen_u64(M) - (a.bits - 1) : 0;
    if (blockIdx.x == 0 && threadIdx.x == 0) *a.out_exp = e0 + r;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t t0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (VEC && NIN > 0) {
        const int64_t nv = a.n / 16;
        const bool w32 = max_shift(a, sh) <= kW32Shift;
        for (int64_t v0 = t0; v0 < nv; v0 += stride * kU) {
            int4 raw[kU][NIN > 0 ? NIN : 1];
#pragma unroll
            for (int u = 0; u < kU; u++) merge_load16<NIN>(a, v0 + u * stride, nv, raw[u]);
#pragma unroll
            for (int u = 0; u < kU; u++) {
                const int64_t v = v0 + u * stride;
                if (v >= nv) break;
                uint32_t w[4] = {0, 0, 0, 0};
                if (w32) {
                    int32_t s[16];
                    merge_sum16_raw<NIN>(a, sh, raw[u], s);
#pragma unroll
                    for (int t = 0; t < 16; t++)
                        w[t >> 2] |= (uint32_t)(uint8_t)sq_code32(s[t], r, a.bits) << (8 * (t & 3));
                } else {
                    int64_t s[16];
                    merge_sum16_raw<NIN>(a, sh, raw[u], s);
#pragma unroll
                    for (int t = 0; t < 16; t++)
                        w[t >> 2] |= (uint32_t)(uint8_t)sq_code(s[t], r, a.bits) << (8 * (t & 3));
                }
                *(int4*)(a.out + v * 16) = make_int4((int)w[0], (int)w[1], (int)w[2], (int)w[3]);
            }
        }
    } else if (VEC) {
        for (int64_t v = t0; v < a.n / 16; v += stride) {
            int64_t s[16];
            merge_sum16(a, sh, v * 16, s);
            uint32_t w[4] = {0, 0, 0, 0};
#pragma unroll
            for (int t = 0; t < 16; t++)
                w[t >> 2] |= (uint32_t)(uint8_t)sq_code(s[t], r, a.bits) << (8 * (t & 3));
            *(int4*)(a.out + v * 16) = make_int4((int)w[0], (int)w[1], (int)w[2], (int)w[3]);
        }
    } else {
        for (int64_t j = t0; j < a.n; j += stride) a.out[j] = (int8_t)sq_code(merge_sum1(a, sh, j), r, a.bits);
    }
}

// pass 2 of a sum whose codes then go through the backward of a ReLU: the
// codes of the sum, zeroed where the exact sum of the mask inputs (m) is not
// positive (the sum's exponent comes from the unmasked max, as when the two
// steps run apart); 16-byte vectors, two inputs on each side
__global__ __launch_bounds__(256) void k_merge_apply_mask(MergeArgs a, MergeArgs m, int64_t nparts)
{
    int sh[kMaxIn], e0, msh[kMaxIn], me0;
    merge_shifts(a, sh, &e0);
    if (!merge_shifts(m, msh, &me0) && blockIdx.x == 0 && threadIdx.x == 0) set_status(a.status, ISEG_DEV_RANGE);
    const uint64_t M = reduce_partials_u64(a.part, nparts);
    const int r = M ? bitlen_u64(M) - (a.bits - 1) : 0;
    if (blockIdx.x == 0 && threadIdx.x == 0) *a.out_exp = e0 + r;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t t0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t nv = a.n / 16;
    const bool w32 = max_shift(a, sh) <= kW32Shift, mw32 = max_shift(m, msh) <= kW32Shift;
    for (int64_t v0 = t0; v0 < nv; v0 += stride * kU) {
        int4 raw[kU][2], mraw[kU][2];
#pragma unroll
        for (int u = 0; u < kU; u++) {
            merge_load16<2>(a, v0 + u * stride, nv, raw[u]);
            merge_load16<2>(m, v0 + u * stride, nv, mraw[u]);
        }
#pragma unroll
        for (int u = 0; u < kU; u++) {
            const int64_t v = v0 + u * stride;
            if (v >= nv) break;
            bool pos[16];
            if (mw32) {
                int32_t ms[16];
                merge_sum16_raw<2>(m, msh, mraw[u], ms);
#pragma unroll
                for (int t = 0; t < 16; t++) pos[t] = ms[t] > 0;
            } else {
                int64_t ms[16];
                merge_sum16_raw<2>(m, msh, mraw[u], ms);
#pragma unroll
                for (int t = 0; t < 16; t++) pos[t] = ms[t] > 0;
            }
            uint32_t w[4] = {0, 0, 0, 0};
            if (w32) {
                int32_t s[16];
                merge_sum16_raw<2>(a, sh, raw[u], s);
#pragma unroll
                for (int t = 0; t < 16; t++)
                    if (pos[t]) w[t >> 2] |= (uint32_t)(uint8_t)sq_code32(s[t], r, a.bits) << (8 * (t & 3));
            } else {
                int64_t s[16];
                merge_sum16_raw<2>(a, sh, raw[u], s);
#pragma unroll
                for (int t = 0; t < 16; t++)
                    if (pos[t]) w[t >> 2] |= (uint32_t)(uint8_t)sq_code(s[t], r, a.bits) << (8 * (t & 3));
            }
            *(int4*)(a.out + v * 16) = make_int4((int)w[0], (int)w[1], (int)w[2], (int)w[3]);
        }
    }
}

// ReLU mask of a merged sum: dx = dy where sum_i a_i 2^e_i > 0, else 0
template <bool VEC, int NIN>
__global__ __launch_bounds__(256) void k_relu_mask(MergeArgs a, const int8_t* __restrict__ dy)
{
    int sh[kMaxIn], e0;
    if (!merge_shifts(a, sh, &e0) && blockIdx.x == 0 && threadIdx.x == 0) set_status(a.status, ISEG_DEV_RANGE);
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t t0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (VEC && NIN > 0) {
        const int64_t nv = a.n / 16;
        const bool w32 = max_shift(a, sh) <= kW32Shift;
        for (int64_t v0 = t0; v0 < nv; v0 += stride * kU) {
          int4 raw[kU][NIN > 0 ? NIN : 1], dr[kU];
#pragma unroll
          for (int u = 0; u < kU; u++) {
              merge_load16<NIN>(a, v0 + u * stride, nv, raw[u]);
              if (v0 + u * stride < nv) dr[u] = *(const int4*)(dy + (v0 + u * stride) * 16);
          }
#pragma unroll
          for (int u = 0; u < kU; u++) {
            const int64_t v = v0 + u * stride;
            if (v >= nv) break;
            const int4 d = dr[u];
            const uint32_t dw[4] = {(uint32_t)d.x, (uint32_t)d.y, (uint32_t)d.z, (uint32_t)d.w};
            uint32_t w[4] = {0, 0, 0, 0};
            if (w32) {
                int32_t s[16];
                merge_sum16_raw<NIN>(a, sh, raw[u], s);
#pragma unroll
                for (int t = 0; t < 16; t++)
                    if (s[t] > 0) w[t >> 2] |= dw[t >> 2] & (0xffu << (8 * (t & 3)));
            } else {
                int64_t s[16];
                merge_sum16_raw<NIN>(a, sh, raw[u], s);
#pragma unroll
                for (int t = 0; t < 16; t++)
                    if (s[t] > 0) w[t >> 2] |= dw[t >> 2] & (0xffu << (8 * (t & 3)));
            }
            *(int4*)(a.out + v * 16) = make_int4((int)w[0], (int)w[1], (int)w[2], (int)w[3]);
          }
        }
    } else if (VEC) {
        for (int64_t v = t0; v < a.n / 16; v += stride) {
            int64_t s[16];
            merge_sum16(a, sh, v * 16, s);
            const int4 d = *(const int4*)(dy + v * 16);
            const uint32_t dw[4] = {(uint32_t)d.x, (uint32_t)d.y, (uint32_t)d.z, (uint32_t)d.w};
            uint32_t w[4] = {0, 0, 0, 0};
#pragma unroll
            for (int t = 0; t < 16; t++)
                if (s[t] > 0) w[t >> 2] |= dw[t >> 2] & (0xffu << (8 * (t & 3)));
            *(int4*)(a.out + v * 16) = make_int4((int)w[0], (int)w[1], (int)w[2], (int)w[3]);
        }
    } else {
        for (int64_t j = t0; j < a.n; j += stride) a.out[j] = merge_sum1(a, sh, j) > 0 ? dy[j] : (int8_t)0;
    }
}

// ---------------------------------------------------------------------------
// concatenation along channels
// ---------------------------------------------------------------------------
struct CatArgs {
    const int8_t* p[kMaxIn];
    const int32_t* e[kMaxIn];
    int32_t off[kMaxIn + 1];       // channel offsets in the output (prefix sums)
    int32_t bc[kMaxIn];
    int32_t n_in;
    int64_t rows, HW;              // rows = N * HW of the output
    int32_t Ctot, bits;
    int32_t blocks_per_part;
    uint64_t* part;                // [n_in][blocks_per_part]
    int8_t* out;
    int32_t* out_exp;
    int32_t* status;
};

__device__ __forceinline__ bool cat_shifts(const CatArgs& a, int* sh, int* e0_out)
{
    int lo = INT_MAX, hi = INT_MIN;
    for (int i = 0; i < a.n_in; i++) {
        lo = *a.e[i] < lo ? *a.e[i] : lo;
        hi = *a.e[i] > hi ? *a.e[i] : hi;
    }
    for (int i = 0; i < a.n_in; i++) {
        const int d = *a.e[i] - lo;
        sh[i] = d > kMaxGap ? kMaxGap : d;
    }
    *e0_out = lo;
    return hi - lo <= kMaxGap;
}

// pass 1: max |code| of each part (blockIdx.y = part)
__global__ __launch_bounds__(256) void k_concat_max(CatArgs a)
{
    const int i = blockIdx.y;
    const int64_t rows_i = a.bc[i] ? a.rows / a.HW : a.rows;
    const int64_t n = rows_i * (a.off[i + 1] - a.off[i]);
    const int8_t* p = a.p[i];
    uint32_t m = 0;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t t0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if ((((uintptr_t)p) & 3) == 0) {
        for (int64_t v = t0; v < n / 4; v += stride) {
            const uint32_t w = *(const uint32_t*)(p + 4 * v);
#pragma unroll
            for (int t = 0; t < 4; t++) {
                const int q = (int8_t)(w >> (8 * t));
                const uint32_t u = (uint32_t)(q < 0 ? -q : q);
                m = u > m ? u : m;
            }
        }
        for (int64_t j = (n / 4) * 4 + t0; j < n; j += stride) {
            const int q = p[j];
            const uint32_t u = (uint32_t)(q < 0 ? -q : q);
            m = u > m ? u : m;
        }
    } else {
        for (int64_t j = t0; j < n; j += stride) {
            const int q = p[j];
            const uint32_t u = (uint32_t)(q < 0 ? -q : q);
            m = u > m ? u : m;
        }
    }
    const uint64_t bm = block_max_u64(m);
    if (threadIdx.x == 0) a.part[(int64_t)i * a.blocks_per_part + blockIdx.x] = bm;
}

template <bool VEC>
__global__ __launch_bounds__(256) void k_concat_apply(CatArgs a)
{
    int sh[kMaxIn], e0;
    const bool ok = cat_shifts(a, sh, &e0);
    // the tensor max is the largest aligned part max
    __shared__ uint64_t pm[kMaxIn];
    for (int i = 0; i < a.n_in; i++) {
        const uint64_t m = reduce_partials_u64(a.part + (int64_t)i * a.blocks_per_part, a.blocks_per_part);
        if (threadIdx.x == 0) pm[i] = m << sh[i];
    }
    __syncthreads();
    uint64_t M = 0;
    for (int i = 0; i < a.n_in; i++) M = pm[i] > M ? pm[i] : M;
    const int r = M ? bitlen_u64(M) - (a.bits - 1) : 0;
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        *a.out_exp = e0 + r;
        if (!ok) set_status(a.status, ISEG_DEV_RANGE);
    }
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t t0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int G = VEC ? 16 : 1;
    const int64_t per_row = a.Ctot / G;
    for (int64_t v = t0; v < a.rows * per_row; v += stride) {
        const int64_t row = v / per_row;
        const int c = (int)(v % per_row) * G;
        int i = 0;
        while (c >= a.off[i + 1]) i++;
        const int Ci = a.off[i + 1] - a.off[i];
        const int64_t srow = a.bc[i] ? row / a.HW : row;
        const int8_t* src = a.p[i] + srow * Ci + (c - a.off[i]);
        if (VEC) {
            const int4 q = *(const int4*)src;
            const int32_t w_in[4] = {q.x, q.y, q.z, q.w};
            uint32_t w[4] = {0, 0, 0, 0};
#pragma unroll
            for (int t = 0; t < 16; t++) {
                const int64_t s = (int64_t)(int8_t)(w_in[t >> 2] >> (8 * (t & 3))) << sh[i];
                w[t >> 2] |= (uint32_t)(uint8_t)sq_code(s, r, a.bits) << (8 * (t & 3));
            }
            *(int4*)(a.out + row * a.Ctot + c) = make_int4((int)w[0], (int)w[1], (int)w[2], (int)w[3]);
        } else {
            a.out[row * a.Ctot + c] = (int8_t)sq_code((int64_t)*src << sh[i], r, a.bits);
        }
    }
}

// backward of the concatenation: channel slices of dy (blockIdx.y = part)
struct SplitArgs {
    int8_t* out[kMaxIn];
    int32_t off[kMaxIn + 1];
    int32_t n_in, Ctot;
    int64_t rows;
    const int8_t* dy;
};

__global__ __launch_bounds__(256) void k_concat_split(SplitArgs a)
{
    const int i = blockIdx.y;
    int8_t* o = a.out[i];
    if (!o) return;
    const int Ci = a.off[i + 1] - a.off[i];
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t t0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const bool vec = (Ci % 16) == 0 && (a.off[i] % 16) == 0 && (a.Ctot % 16) == 0 &&
                     ((((uintptr_t)a.dy) | (uintptr_t)o) & 15) == 0;
    if (vec) {
        const int64_t per_row = Ci / 16;
        for (int64_t v = t0; v < a.rows * per_row; v += stride) {
            const int64_t row = v / per_row;
            const int c = (int)(v % per_row) * 16;
            *(int4*)(o + row * Ci + c) = *(const int4*)(a.dy + row * a.Ctot + a.off[i] + c);
        }
    } else {
        for (int64_t j = t0; j < a.rows * Ci; j += stride) {
            const int64_t row = j / Ci;
            const int c = (int)(j % Ci);
            o[j] = a.dy[row * a.Ctot + a.off[i] + c];
        }
    }
}

// ---------------------------------------------------------------------------
// spatial means: out[n, c] = SQ(sum_hw x[n, hw, c0 + c] / divisor)
// ---------------------------------------------------------------------------
struct SsumArgs {
    const int8_t* x;
    int64_t N, HW, ldc, c0, C;
    int64_t rows_per_split;
    int32_t splits;
    int32_t* part;                 // [splits][N][C] int32 partial sums
    int64_t* sums;                 // [N][C] exact sums
    uint64_t* pmax;                // max |sum| partials, one per reduce block
    const int32_t* x_exp;
    int64_t divisor;
    int32_t bits;
    int8_t* out;
    int32_t* out_exp;
};

// block (image n, 256-channel chunk, hw split): 64 lanes x 4 channels, the
// four waves take interleaved rows; fixed-order combine through LDS
__global__ __launch_bounds__(256) void k_ssum_part4(SsumArgs a)
{
    __shared__ int32_t red[4][256];
    const int64_t nchunk = (a.C + 255) / 256;
    const int64_t n = blockIdx.x / nchunk;
    const int64_t cbase = (blockIdx.x % nchunk) * 256;
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int64_t c = cbase + 4 * lane;
    const int64_t h0 = (int64_t)blockIdx.y * a.rows_per_split;
    int64_t h1 = h0 + a.rows_per_split;
    h1 = h1 < a.HW ? h1 : a.HW;
    int32_t s[4] = {0, 0, 0, 0};
    if (c < a.C) {
        const int8_t* base = a.x + n * a.HW * a.ldc + a.c0 + c;
        for (int64_t h = h0 + wv; h < h1; h += 4) {
            const uint32_t w = *(const uint32_t*)(base + h * a.ldc);
#pragma unroll
            for (int t = 0; t < 4; t++) s[t] += (int8_t)(w >> (8 * t));
        }
    }
#pragma unroll
    for (int t = 0; t < 4; t++) red[wv][4 * lane + t] = s[t];
    __syncthreads();
    const int cc = threadIdx.x;
    if (cbase + cc < a.C) {
        const int32_t v = red[0][cc] + red[1][cc] + red[2][cc] + red[3][cc];
        a.part[((int64_t)blockIdx.y * a.N + n) * a.C + cbase + cc] = v;
    }
}

// any layout: one lane per channel
__global__ __launch_bounds__(256) void k_ssum_part1(SsumArgs a)
{
    const int64_t nchunk = (a.C + 255) / 256;
    const int64_t n = blockIdx.x / nchunk;
    const int64_t c = (blockIdx.x % nchunk) * 256 + threadIdx.x;
    if (c >= a.C) return;
    const int64_t h0 = (int64_t)blockIdx.y * a.rows_per_split;
    int64_t h1 = h0 + a.rows_per_split;
    h1 = h1 < a.HW ? h1 : a.HW;
    int32_t s = 0;
    const int8_t* base = a.x + n * a.HW * a.ldc + a.c0 + c;
    for (int64_t h = h0; h < h1; h++) s += base[h * a.ldc];
    a.part[((int64_t)blockIdx.y * a.N + n) * a.C + c] = s;
}

// exact int64 sum of each (n, c)'s split partials: a block takes 64 elements,
// its four waves a quarter of the splits each (four loads in flight per lane),
// the wave sums added through LDS; per-block max |sum| partials
__global__ __launch_bounds__(256) void k_ssum_reduce(SsumArgs a)
{
    __shared__ int64_t red[4][64];
    const int64_t nc = a.N * a.C;
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int64_t j = (int64_t)blockIdx.x * 64 + lane;
    int64_t s = 0;
    if (j < nc) {
        int k = wv;
        for (; k + 12 < a.splits; k += 16) {
            const int32_t v0 = a.part[(int64_t)k * nc + j], v1 = a.part[(int64_t)(k + 4) * nc + j];
            const int32_t v2 = a.part[(int64_t)(k + 8) * nc + j], v3 = a.part[(int64_t)(k + 12) * nc + j];
            s += ((int64_t)v0 + v1) + ((int64_t)v2 + v3);
        }
        for (; k < a.splits; k += 4) s += a.part[(int64_t)k * nc + j];
    }
    red[wv][lane] = s;
    __syncthreads();
    uint64_t m = 0;
    if (wv == 0 && j < nc) {
        const int64_t t = red[0][lane] + red[1][lane] + red[2][lane] + red[3][lane];
        a.sums[j] = t;
        m = (uint64_t)(t < 0 ? -t : t);
    }
    block_store_max_u64(m, a.pmax);
}

// SQ of sum / D.  With u the smallest integer such that max|sum| < D 2^u
// (the max from the reduce blocks' partials), the scale is 2^(x_exp + u) and
// code = floor(sum 2^(bits-1-u) / D + 1/2), decided exactly.
__global__ __launch_bounds__(256) void k_ssum_code(SsumArgs a, int64_t nparts)
{
    const int64_t nc = a.N * a.C;
    const uint64_t M = nparts ? reduce_partials_u64(a.pmax, nparts) : 0;
    const i128 D = a.divisor;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    if (M == 0) {
        if (blockIdx.x == 0 && threadIdx.x == 0) *a.out_exp = *a.x_exp - bitlen_u64((uint64_t)(a.divisor - 1));
        for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < nc; j += stride) a.out[j] = 0;
        return;
    }
    const int u = ceil_pow2_exp128((i128)M, D);
    const int sh = a.bits - 1 - u;
    if (blockIdx.x == 0 && threadIdx.x == 0) *a.out_exp = *a.x_exp + u + 1 - a.bits;
    for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < nc; j += stride)
        a.out[j] = (int8_t)clamp_k128(rhu128(a.sums[j], sh, D), a.bits);
}

bool fill_merge_inputs(MergeArgs& m, int32_t n_in, const int8_t* const* in, const int32_t* const* in_exp,
                       const int32_t* exp_add, const int32_t* bcast)
{
    if (n_in < 1 || n_in > kMaxIn || !in || !in_exp) return false;
    m.n_in = n_in;
    for (int i = 0; i < n_in; i++) {
        if (!in_exp[i]) return false;
        m.p[i] = in[i];
        m.e[i] = in_exp[i];
        m.add[i] = exp_add ? exp_add[i] : 0;
        m.bc[i] = bcast ? (bcast[i] != 0) : 0;
        if (m.add[i] < -256 || m.add[i] > 256) return false;
    }
    m.any_bc = 0;
    for (int i = 0; i < n_in; i++) m.any_bc |= m.bc[i];
    return true;
}

}  // namespace

// ---------------------------------------------------------------------------
// C ABI
// ---------------------------------------------------------------------------
extern "C" size_t iseg_sum_requant_ws(int64_t, int64_t, int64_t) { return align256(kMaxPartials * 8); }

extern "C" int iseg_sum_requant(int32_t n_in, const int8_t* const* in, const int32_t* const* in_exp,
                                const int32_t* exp_add, const int32_t* bcast, int64_t N, int64_t HW, int64_t C,
                                int32_t relu, int32_t bits, int8_t* out, int32_t* out_exp, void* ws,
                                size_t ws_bytes, int32_t* dev_status, hipStream_t stream)
{
    MergeArgs a{};
    if (!fill_merge_inputs(a, n_in, in, in_exp, exp_add, bcast)) return ISEG_ERR_ARG;
    if (N < 0 || HW < 0 || C < 0 || bits < 2 || bits > 8 || !out_exp) return ISEG_ERR_ARG;
    const int64_t n = N * HW * C;
    if (n > 0 && !out) return ISEG_ERR_ARG;
    for (int i = 0; i < n_in; i++)
        if (n > 0 && !in[i]) return ISEG_ERR_ARG;
    if (!ws || ws_bytes < iseg_sum_requant_ws(N, HW, C)) return ISEG_ERR_WORKSPACE;
    a.n = n; a.HW = HW; a.C = C; a.relu = relu != 0; a.bits = bits;
    a.part = (uint64_t*)ws; a.out = out; a.out_exp = out_exp; a.status = dev_status;
    bool vec = (C % 16) == 0 && ((uintptr_t)out & 15) == 0;
    for (int i = 0; i < n_in; i++) vec = vec && (((uintptr_t)in[i]) & 15) == 0;
    const int64_t units = vec ? n / 16 : n;
    const unsigned g1 = grid_for(units, 256 * kU, kMaxPartials);
    const bool two = n_in == 2;
    if (vec && two) hipLaunchKernelGGL((k_merge_max<true, 2>), dim3(g1), dim3(256), 0, stream, a);
    else if (vec) hipLaunchKernelGGL((k_merge_max<true, 0>), dim3(g1), dim3(256), 0, stream, a);
    else hipLaunchKernelGGL((k_merge_max<false, 0>), dim3(g1), dim3(256), 0, stream, a);
    int rc = launch_ok();
    if (rc) return rc;
    const unsigned g2 = grid_for(units, 256 * kU, 1024);
    if (vec && two) hipLaunchKernelGGL((k_merge_apply<true, 2>), dim3(g2), dim3(256), 0, stream, a, (int64_t)g1);
    else if (vec) hipLaunchKernelGGL((k_merge_apply<true, 0>), dim3(g2), dim3(256), 0, stream, a, (int64_t)g1);
    else hipLaunchKernelGGL((k_merge_apply<false, 0>), dim3(g2), dim3(256), 0, stream, a, (int64_t)g1);
    return launch_ok();
}

extern "C" int iseg_sum_requant_relu_mask(int32_t n_in, const int8_t* const* in, const int32_t* const* in_exp,
                                          const int32_t* exp_add, int64_t N, int64_t HW, int64_t C, int32_t bits,
                                          int32_t n_mask, const int8_t* const* mask_in,
                                          const int32_t* const* mask_exp, int8_t* out, int32_t* out_exp, void* ws,
                                          size_t ws_bytes, int32_t* dev_status, hipStream_t stream)
{
    MergeArgs a{}, m{};
    if (!fill_merge_inputs(a, n_in, in, in_exp, exp_add, nullptr)) return ISEG_ERR_ARG;
    if (!fill_merge_inputs(m, n_mask, mask_in, mask_exp, nullptr, nullptr)) return ISEG_ERR_ARG;
    if (N < 0 || HW < 0 || C < 1 || bits < 2 || bits > 8 || !out_exp) return ISEG_ERR_ARG;
    const int64_t n = N * HW * C;
    if (n > 0 && !out) return ISEG_ERR_ARG;
    for (int i = 0; i < n_in; i++)
        if (n > 0 && !in[i]) return ISEG_ERR_ARG;
    for (int i = 0; i < n_mask; i++)
        if (n > 0 && !mask_in[i]) return ISEG_ERR_ARG;
    if (!ws || ws_bytes < iseg_sum_requant_ws(N, HW, C)) return ISEG_ERR_WORKSPACE;
    bool vec = n_in == 2 && n_mask == 2 && (C % 16) == 0 && ((uintptr_t)out & 15) == 0;
    for (int i = 0; i < n_in; i++) vec = vec && (((uintptr_t)in[i]) & 15) == 0;
    for (int i = 0; i < n_mask; i++) vec = vec && (((uintptr_t)mask_in[i]) & 15) == 0;
    if (!vec) {
        // the two steps apart (the mask pass in place on the codes)
        int rc = iseg_sum_requant(n_in, in, in_exp, exp_add, nullptr, N, HW, C, 0, bits, out, out_exp, ws, ws_bytes,
                                  dev_status, stream);
        if (rc) return rc;
        return iseg_relu_mask_bwd(out, n_mask, mask_in, mask_exp, nullptr, n, C, out, dev_status, stream);
    }
    a.n = n; a.HW = HW; a.C = C; a.relu = 0; a.bits = bits;
    a.part = (uint64_t*)ws; a.out = out; a.out_exp = out_exp; a.status = dev_status;
    m.n = n; m.HW = HW; m.C = C;
    const int64_t units = n / 16;
    const unsigned g1 = grid_for(units, 256 * kU, kMaxPartials);
    hipLaunchKernelGGL((k_merge_max<true, 2>), dim3(g1), dim3(256), 0, stream, a);
    int rc = launch_ok();
    if (rc) return rc;
    const unsigned g2 = grid_for(units, 256 * kU, 1024);
    hipLaunchKernelGGL(k_merge_apply_mask, dim3(g2), dim3(256), 0, stream, a, m, (int64_t)g1);
    return launch_ok();
}

extern "C" int iseg_relu_mask_bwd(const int8_t* dy, int32_t n_in, const int8_t* const* in,
                                  const int32_t* const* in_exp, const int32_t* exp_add, int64_t n, int64_t C,
                                  int8_t* dx, int32_t* dev_status, hipStream_t stream)
{
    MergeArgs a{};
    if (!fill_merge_inputs(a, n_in, in, in_exp, exp_add, nullptr)) return ISEG_ERR_ARG;
    if (n < 0 || C < 1 || n % C != 0) return ISEG_ERR_ARG;
    if (n > 0 && (!dy || !dx)) return ISEG_ERR_ARG;
    for (int i = 0; i < n_in; i++)
        if (n > 0 && !in[i]) return ISEG_ERR_ARG;
    if (n == 0) return ISEG_OK;
    bool vec = (C % 16) == 0 && ((((uintptr_t)dy) | (uintptr_t)dx) & 15) == 0;
    for (int i = 0; i < n_in; i++) vec = vec && (((uintptr_t)in[i]) & 15) == 0;
    a.n = n; a.HW = n / C; a.C = C;
    a.out = dx; a.status = dev_status;
    const dim3 grid(grid_for(vec ? n / 16 : n, vec ? 256 * kU : 256, 2048));
    if (vec && n_in == 2) hipLaunchKernelGGL((k_relu_mask<true, 2>), grid, dim3(256), 0, stream, a, dy);
    else if (vec) hipLaunchKernelGGL((k_relu_mask<true, 0>), grid, dim3(256), 0, stream, a, dy);
    else hipLaunchKernelGGL((k_relu_mask<false, 0>), grid, dim3(256), 0, stream, a, dy);
    return launch_ok();
}

extern "C" size_t iseg_concat_requant_ws(int32_t n_in) { return align256((size_t)(n_in > 0 ? n_in : 1) * 64 * 8); }

extern "C" int iseg_concat_requant(int32_t n_in, const int8_t* const* in, const int32_t* const* in_exp,
                                   const int64_t* C_in, const int32_t* bcast, int64_t N, int64_t HW, int32_t bits,
                                   int8_t* out, int32_t* out_exp, void* ws, size_t ws_bytes, int32_t* dev_status,
                                   hipStream_t stream)
{
    CatArgs a{};
    if (n_in < 1 || n_in > kMaxIn || !in || !in_exp || !C_in || !out_exp) return ISEG_ERR_ARG;
    if (N < 0 || HW < 1 || bits < 2 || bits > 8) return ISEG_ERR_ARG;
    if (!ws || ws_bytes < iseg_concat_requant_ws(n_in)) return ISEG_ERR_WORKSPACE;
    a.n_in = n_in;
    a.off[0] = 0;
    bool vec = ((uintptr_t)out & 15) == 0;
    for (int i = 0; i < n_in; i++) {
        if (!in_exp[i] || C_in[i] < 1 || (N > 0 && !in[i])) return ISEG_ERR_ARG;
        a.p[i] = in[i];
        a.e[i] = in_exp[i];
        a.bc[i] = bcast ? (bcast[i] != 0) : 0;
        if ((int64_t)a.off[i] + C_in[i] > (1 << 24)) return ISEG_ERR_UNSUPPORTED;
        a.off[i + 1] = a.off[i] + (int32_t)C_in[i];
        vec = vec && (C_in[i] % 16) == 0 && (((uintptr_t)in[i]) & 15) == 0;
    }
    if (N > 0 && !out) return ISEG_ERR_ARG;
    a.rows = N * HW; a.HW = HW; a.Ctot = a.off[n_in]; a.bits = bits;
    a.blocks_per_part = 64;
    a.part = (uint64_t*)ws; a.out = out; a.out_exp = out_exp; a.status = dev_status;
    hipLaunchKernelGGL(k_concat_max, dim3(a.blocks_per_part, n_in), dim3(256), 0, stream, a);
    int rc = launch_ok();
    if (rc) return rc;
    const int64_t units = a.rows * a.Ctot / (vec ? 16 : 1);
    if (vec) hipLaunchKernelGGL(k_concat_apply<true>, dim3(grid_for(units, 256, 2048)), dim3(256), 0, stream, a);
    else hipLaunchKernelGGL(k_concat_apply<false>, dim3(grid_for(units, 256, 2048)), dim3(256), 0, stream, a);
    return launch_ok();
}

extern "C" int iseg_concat_split(const int8_t* dy, int64_t rows, int32_t n_in, const int64_t* C_in,
                                 int8_t* const* out, hipStream_t stream)
{
    SplitArgs a{};
    if (n_in < 1 || n_in > kMaxIn || !C_in || !out || rows < 0) return ISEG_ERR_ARG;
    a.off[0] = 0;
    for (int i = 0; i < n_in; i++) {
        if (C_in[i] < 1 || (int64_t)a.off[i] + C_in[i] > (1 << 24)) return ISEG_ERR_ARG;
        a.out[i] = out[i];
        a.off[i + 1] = a.off[i] + (int32_t)C_in[i];
    }
    if (rows > 0 && !dy) return ISEG_ERR_ARG;
    if (rows == 0) return ISEG_OK;
    a.n_in = n_in; a.Ctot = a.off[n_in]; a.rows = rows; a.dy = dy;
    const int64_t units = rows * a.Ctot / 16 + 1;
    hipLaunchKernelGGL(k_concat_split, dim3(grid_for(units / n_in + 1, 256, 2048), n_in), dim3(256), 0, stream, a);
    return launch_ok();
}

static int64_t ssum_splits(int64_t N, int64_t HW, int64_t C)
{
    const int64_t blocks = N * ((C + 255) / 256);
    int64_t s = blocks > 0 ? 512 / blocks : 1;
    if (s < 1) s = 1;
    if (s > HW) s = HW;
    if (s > 1024) s = 1024;
    return s < 1 ? 1 : s;
}

extern "C" size_t iseg_spatial_sum_ws(int64_t N, int64_t HW, int64_t C)
{
    const int64_t s = ssum_splits(N, HW, C);
    return align256((size_t)(s * N * C) * 4) + align256((size_t)(N * C) * 8) +
           align256((size_t)ceil_div64(N * C, 64) * 8);
}

extern "C" int iseg_spatial_sum(const int8_t* x, const int32_t* x_exp, int64_t N, int64_t HW, int64_t ldc,
                                int64_t c0, int64_t C, int64_t divisor, int32_t bits, int8_t* out,
                                int32_t* out_exp, void* ws, size_t ws_bytes, int32_t* dev_status,
                                hipStream_t stream)
{
    (void)dev_status;
    if (N < 0 || HW < 1 || C < 1 || c0 < 0 || c0 + C > ldc || bits < 2 || bits > 8) return ISEG_ERR_ARG;
    if (!x_exp || !out_exp || (N > 0 && (!x || !out))) return ISEG_ERR_ARG;
    if (divisor < 1 || divisor > (1 << 30)) return ISEG_ERR_ARG;
    if (HW > (1 << 23) || N * C > (1 << 20)) return ISEG_ERR_UNSUPPORTED;
    if (!ws || ws_bytes < iseg_spatial_sum_ws(N, HW, C)) return ISEG_ERR_WORKSPACE;
    SsumArgs a{};
    a.x = x; a.N = N; a.HW = HW; a.ldc = ldc; a.c0 = c0; a.C = C;
    a.splits = (int32_t)ssum_splits(N, HW, C);
    a.rows_per_split = ceil_div64(HW, a.splits);
    a.splits = (int32_t)ceil_div64(HW, a.rows_per_split);
    a.part = (int32_t*)ws;
    a.sums = (int64_t*)((char*)ws + align256((size_t)(a.splits * N * C) * 4));
    a.pmax = (uint64_t*)((char*)a.sums + align256((size_t)(N * C) * 8));
    a.x_exp = x_exp; a.divisor = divisor; a.bits = bits; a.out = out; a.out_exp = out_exp;
    if (N > 0) {
        dim3 grid((unsigned)(N * ((C + 255) / 256)), (unsigned)a.splits);
        const bool v4 = (ldc % 4) == 0 && (c0 % 4) == 0 && (C % 4) == 0 && (((uintptr_t)x) & 3) == 0;
        if (v4) hipLaunchKernelGGL(k_ssum_part4, grid, dim3(256), 0, stream, a);
        else hipLaunchKernelGGL(k_ssum_part1, grid, dim3(256), 0, stream, a);
        int rc = launch_ok();
        if (rc) return rc;
    }
    const int64_t nred = ceil_div64(N * C, 64);
    if (nred > 0) {
        hipLaunchKernelGGL(k_ssum_reduce, dim3((unsigned)nred), dim3(256), 0, stream, a);
        int rc = launch_ok();
        if (rc) return rc;
    }
    hipLaunchKernelGGL(k_ssum_code, dim3(grid_for(N * C, 256, 256)), dim3(256), 0, stream, a, nred);
    return launch_ok();
}
