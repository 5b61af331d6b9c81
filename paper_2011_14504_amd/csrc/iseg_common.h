// iseg_common.h -- device/host helpers shared by the libiseg kernels.
//
// Exact integer arithmetic (bit lengths, floor division, half-up rounding of
// rationals scaled by powers of two), the Philox4x32-10 block, 64-wide wave
// reductions and the small launch helpers.  The one use of floating point is a
// quotient estimate inside floordiv128 that an integer remainder check makes
// exact.
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>
#include <stdint.h>

#include "iseg.h"

typedef __int128 i128;
typedef unsigned __int128 u128;

#define ISEG_HD __host__ __device__ __forceinline__

// ---------------------------------------------------------------------------
// bit lengths and powers of two
// ---------------------------------------------------------------------------
ISEG_HD int bitlen_u64(uint64_t v) { return v ? 64 - __builtin_clzll(v) : 0; }

ISEG_HD int bitlen_u128(u128 v)
{
    uint64_t hi = (uint64_t)(v >> 64);
    return hi ? 64 + bitlen_u64(hi) : bitlen_u64((uint64_t)v);
}

ISEG_HD i128 abs128(i128 v) { return v < 0 ? -v : v; }
ISEG_HD int bitlen_i128(i128 v) { return bitlen_u128((u128)abs128(v)); }
ISEG_HD i128 pow2_128(int e) { return (i128)1 << e; }

// double of an i128 up to two roundings of its magnitude (relative error
// < 2^-51; the halves of |v| are both non-negative, so nothing cancels)
ISEG_HD double i128_to_double(i128 v)
{
    const u128 m = (u128)(v < 0 ? -v : v);
    const double d = (double)(uint64_t)(m >> 64) * 18446744073709551616.0 + (double)(uint64_t)m;
    return v < 0 ? -d : d;
}

// floor(a / b) for b > 0, exact.  When |a| / b < 2^48 (bit lengths differ by
// less than 48) the double quotient is off the true one by less than 0.2, so
// its floor is within one of floor(a / b) and the integer remainder check
// settles it; only larger quotients take the software 128-bit divide (a long
// loop on the GPU, which has no integer divide instruction).
ISEG_HD i128 floordiv128(i128 a, i128 b)
{
    if (bitlen_i128(a) - bitlen_i128(b) < 48) {
        i128 q = (i128)(int64_t)floor(i128_to_double(a) / i128_to_double(b));
        i128 r = a - q * b;
        for (int i = 0; i < 2 && r < 0; i++) { q -= 1; r += b; }
        for (int i = 0; i < 2 && r >= b; i++) { q += 1; r -= b; }
        return q;
    }
    i128 q = a / b;
    if ((a % b) != 0 && a < 0) q -= 1;
    return q;
}

// floor(num * 2^sh / den + 1/2), den > 0 (Eq. 2's half-up rounding)
ISEG_HD i128 rhu128(i128 num, int sh, i128 den)
{
    if (sh >= 0) return floordiv128(2 * (num << sh) + den, 2 * den);
    return floordiv128(2 * num + (den << -sh), 2 * (den << -sh));
}

// A < B * 2^t for A >= 0, B > 0
ISEG_HD bool lt_scaled128(i128 A, i128 B, int t)
{
    return t >= 0 ? A < (B << t) : (A << -t) < B;
}

// smallest e with A < B * 2^e (A > 0, B > 0).  bitlen(A) - bitlen(B) is
// within one of the answer, so each loop runs at most twice.
ISEG_HD int ceil_pow2_exp128(i128 A, i128 B)
{
    int e = bitlen_i128(A) - bitlen_i128(B);
    for (int i = 0; i < 4 && !lt_scaled128(A, B, e); i++) e++;
    for (int i = 0; i < 4 && lt_scaled128(A, B, e - 1); i++) e--;
    return e;
}

ISEG_HD int64_t clamp_k(int64_t v, int k)
{
    int64_t lim = ((int64_t)1 << (k - 1)) - 1;
    return v > lim ? lim : (v < -lim ? -lim : v);
}

ISEG_HD i128 clamp_k128(i128 v, int k)
{
    i128 lim = pow2_128(k - 1) - 1;
    return v > lim ? lim : (v < -lim ? -lim : v);
}

// half-up rounding of q / 2^r for r >= 1 (arithmetic shift = floor)
ISEG_HD int64_t shr_rhu(int64_t q, int r) { return (q + ((int64_t)1 << (r - 1))) >> r; }

// SQ code of an integer for a given shift r (r <= 0: exact left shift)
ISEG_HD int64_t sq_code(int64_t q, int r, int k)
{
    return clamp_k(r > 0 ? shr_rhu(q, r) : q * ((int64_t)1 << -r), k);
}

// ---------------------------------------------------------------------------
// Philox4x32-10 (Salmon et al., SC'11): multipliers 0xD2511F53, 0xCD9E8D57;
// key schedule increments 0x9E3779B9, 0xBB67AE85; ten rounds.
// ---------------------------------------------------------------------------
struct philox_out { uint32_t v[4]; };

ISEG_HD philox_out philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                 uint32_t k0, uint32_t k1)
{
#pragma unroll
    for (int i = 0; i < 10; i++) {
        uint64_t a = (uint64_t)0xD2511F53u * c0;
        uint64_t b = (uint64_t)0xCD9E8D57u * c2;
        uint32_t n0 = (uint32_t)(b >> 32) ^ c1 ^ k0;
        uint32_t n2 = (uint32_t)(a >> 32) ^ c3 ^ k1;
        c1 = (uint32_t)b;
        c3 = (uint32_t)a;
        c0 = n0;
        c2 = n2;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    philox_out o;
    o.v[0] = c0; o.v[1] = c1; o.v[2] = c2; o.v[3] = c3;
    return o;
}

// 64-bit uniform draw of element idx: key (seed, tensor_id), counter (idx, step)
ISEG_HD uint64_t philox_draw(uint64_t seed, uint32_t tensor_id, uint32_t step, uint64_t idx)
{
    philox_out o = philox4x32_10((uint32_t)idx, (uint32_t)(idx >> 32), step, 0u,
                                 (uint32_t)seed, tensor_id);
    return (uint64_t)o.v[0] | ((uint64_t)o.v[1] << 32);
}

// RQ code of an integer (Eq. 5-6): r >= 1 stochastic, r <= 0 exact
ISEG_HD int64_t rq_code(int64_t q, int r, int k, uint64_t draw)
{
    if (r <= 0) return clamp_k(q * ((int64_t)1 << -r), k);
    int64_t fl = q >> r;
    uint64_t rem = (uint64_t)(q & (((int64_t)1 << r) - 1));
    uint64_t ur = draw >> (64 - r);
    return clamp_k(fl + (ur < rem ? 1 : 0), k);
}

// ---------------------------------------------------------------------------
// wave (64 lanes) and block reductions
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        uint32_t t = __shfl_xor(v, o, 64);
        v = t > v ? t : v;
    }
    return v;
}

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        uint64_t t = __shfl_xor(v, o, 64);
        v = t > v ? t : v;
    }
    return v;
}

// block-wide max of a u64, one atomicMax per block into *dst
__device__ __forceinline__ void block_atomic_max_u64(uint64_t v, unsigned long long* dst)
{
    __shared__ uint64_t red[16];
    v = wave_max_u64(v);
    int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    if (lane == 0) red[wid] = v;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint64_t m = 0;
        int nw = (blockDim.x + 63) >> 6;
        for (int i = 0; i < nw; i++) m = red[i] > m ? red[i] : m;
        if (m) atomicMax(dst, (unsigned long long)m);
    }
}

// Device-scope atomics to one address serialize across the chip (several ns
// each), so grid-wide maxima are formed from per-block partials instead:
// block b stores its maximum into part[b] and the consumer reduces them.
__device__ __forceinline__ uint64_t block_max_u64(uint64_t v)
{
    __shared__ uint64_t red_bm[16];
    v = wave_max_u64(v);
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    __syncthreads();                      // red_bm may still be read by a previous call
    if (lane == 0) red_bm[wid] = v;
    __syncthreads();
    uint64_t m = 0;
    const int nw = (blockDim.x + 63) >> 6;
    for (int i = 0; i < nw; i++) m = red_bm[i] > m ? red_bm[i] : m;
    return m;
}

// block max of v stored (plain store) into part[linear block index]
__device__ __forceinline__ void block_store_max_u64(uint64_t v, uint64_t* part)
{
    const uint64_t m = block_max_u64(v);
    if (threadIdx.x == 0) part[(int64_t)blockIdx.y * gridDim.x + blockIdx.x] = m;
}

// max over n partials, computed by the whole block (every thread gets it).
// The loads are unconditional (an index past the end re-reads partial 0, a
// value already in the max) so the eight of a thread are in flight together;
// a guarded load would be compiled as a branch with a wait after each.
__device__ __forceinline__ uint64_t reduce_partials_u64(const uint64_t* part, int64_t n)
{
    uint64_t m = 0;
    for (int64_t base = 0; base < n; base += 8 * (int64_t)blockDim.x) {
        uint64_t v[8];
#pragma unroll
        for (int k = 0; k < 8; k++) {
            const int64_t i = base + k * (int64_t)blockDim.x + threadIdx.x;
            v[k] = part[i < n ? i : 0];
        }
#pragma unroll
        for (int k = 0; k < 8; k++) m = v[k] > m ? v[k] : m;
    }
    return block_max_u64(m);
}

__device__ __forceinline__ void set_status(int32_t* st, int32_t bits)
{
    if (st) atomicOr(st, bits);
}

// ---------------------------------------------------------------------------
// host helpers
// ---------------------------------------------------------------------------
static inline size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

static inline int launch_ok() { return hipGetLastError() == hipSuccess ? ISEG_OK : ISEG_ERR_DEVICE; }

static inline int64_t ceil_div64(int64_t a, int64_t b) { return (a + b - 1) / b; }

// grid size for a grid-stride loop over n items with `per_block` items per block
static inline unsigned grid_for(int64_t n, int64_t per_block, unsigned cap = 4096)
{
    int64_t g = ceil_div64(n > 0 ? n : 1, per_block);
    if (g > cap) g = cap;
    if (g < 1) g = 1;
    return (unsigned)g;
}

// Fill kernel used instead of hipMemsetAsync so the calls stay safe inside
// captured graphs.
__global__ void k_fill_u32(uint32_t* p, int64_t n, uint32_t v);

// device-side requant of an integer buffer whose max |.| is already in *maxp;
// the input exponent is *exp_a + *exp_b + exp_add (NULL pointers count as 0)
// tiling of an int16-staged [rows][cols] conv output: row tiles are runs of
// tile_rows rows (th == 0) or th x tw pixel tiles of Ho x Wo images
struct StageMap {
    int32_t tile_rows, tile_cols;
    int32_t Ho, Wo, th, tw, tiles_y, tiles_x;
};
// requant of int16-staged conv sums (per-tile shifts) to int8 SQ codes
// the tensor max comes from *maxp, or (maxp == NULL) from nparts per-block
// partials that every block of the requant kernel reduces itself
int launch_requant_staged16(const int16_t* in, const uint8_t* tshift, int64_t rows, int32_t cols,
                            const StageMap& sm, const int32_t* exp_a, const int32_t* exp_b, int bits,
                            int8_t* out, int32_t* out_exp, const unsigned long long* maxp, hipStream_t s,
                            const uint64_t* part = nullptr, int64_t nparts = 0);
int launch_requant_apply(const void* in, int in_dtype, int64_t n, const int32_t* exp_a,
                         const int32_t* exp_b, int32_t exp_add, int bits, int stochastic,
                         int keep_scale,
                         uint64_t seed, uint32_t tensor_id, uint32_t step,
                         int out_dtype, void* out, int32_t* out_exp,
                         const unsigned long long* maxp, hipStream_t s,
                         const uint64_t* part = nullptr, int64_t nparts = 0);
// SQ / RQ of the sum of `splits` (<= 8) int32 partial tensors [splits][n]
// (n % 4 == 0, 16-byte aligned partials) into int8 codes; the max from the
// npmax max partials in pmax
int launch_requant_splits(const int32_t* part, int splits, int64_t n, const int32_t* exp_a, const int32_t* exp_b,
                          int bits, int stochastic, int keep_scale, uint64_t seed, uint32_t tensor_id, uint32_t step,
                          int8_t* out, int32_t* out_exp, hipStream_t s, const uint64_t* pmax, int64_t npmax);

// max |.| of an int32/int64 buffer into *maxp (which must be zeroed first)
int launch_absmax(const void* in, int in_dtype, int64_t n, unsigned long long* maxp,
                  int32_t* dev_status, hipStream_t s);

int launch_fill_u32(void* p, int64_t n_words, uint32_t v, hipStream_t s);
// raise a kernel's dynamic LDS limit (cached per device and kernel)
bool lds_limit(const void* f, size_t bytes);
// *maxp = max over n block partials (one block)
int launch_reduce_max(const uint64_t* part, int64_t n, unsigned long long* maxp, hipStream_t s);

// measurement hook (iseg_profile_arm).  prof_claim takes the armed hook for
// one launch (at most one launch ever claims one arming) and hands out its
// two events; prof_begin claims it and records the start event, returning the
// stop event to record after the work, or nullptr.
bool prof_claim(int kid, hipEvent_t* start, hipEvent_t* stop);
hipEvent_t prof_begin(int kid, hipStream_t s);
void prof_end(hipEvent_t stop, hipStream_t s);

// One kernel launch under the hook: when armed, the events are attached to
// the dispatch itself (hipExtLaunchKernelGGL), so they carry the kernel's own
// start and end times, without the queue markers of separate event records.
template <typename F, typename... A>
void timed_launch(int kid, F kernel, const dim3& grid, const dim3& block, uint32_t shmem, hipStream_t s, A... args)
{
    hipEvent_t start = nullptr, stop = nullptr;
    if (prof_claim(kid, &start, &stop))
        hipExtLaunchKernelGGL(kernel, grid, block, shmem, s, start, stop, 0, args...);
    else
        hipLaunchKernelGGL(kernel, grid, block, shmem, s, args...);
}
#define ISEG_TIMED_LAUNCH(kid, stream, ...) timed_launch((kid), __VA_ARGS__)

// measurement hook around a whole entry-point call (every kernel it enqueues)
struct ProfScope {
    hipStream_t s;
    hipEvent_t stop;
    ProfScope(int k, hipStream_t st) : s(st), stop(prof_begin(k, st)) {}
    ~ProfScope()
    {
        if (stop) prof_end(stop, s);
    }
};

// name of the kernel path the calling thread's last convolution entry point
// took (iseg_conv_last_plan); set by the dispatch, per thread
void conv_plan_set(const char* name);
