// profile.hip -- the in-place kernel timing hook (iseg_profile_arm), the
// per-thread record of the convolution path taken (iseg_conv_last_plan), and
// the device status word utilities.
#include <atomic>
#include <mutex>

#include "iseg_common.h"

namespace {
// the armed kernel family; the events belong to the caller.  A launch claims
// the arming under the mutex, so concurrent launches never share one.
std::mutex g_mu;
std::atomic<int> g_kid{ISEG_KID_NONE};
hipEvent_t g_start = nullptr, g_stop = nullptr;

thread_local const char* t_conv_plan = "none";

__global__ void k_status_zero(int32_t* st) { *st = 0; }

__global__ __launch_bounds__(256) void k_check_codes(const int8_t* __restrict__ x, int64_t n, int lim,
                                                     int32_t* dev_status)
{
    bool bad = false;
    const int64_t n16 = n / 16;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += stride) {
        const int4 v = ((const int4*)x)[i];
        const int w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int j = 0; j < 4; j++)
#pragma unroll
            for (int b = 0; b < 4; b++) {
                const int c = (int)(int8_t)(w[j] >> (8 * b));
                bad |= c > lim || c < -lim;
            }
    }
    for (int64_t i = n16 * 16 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
        const int c = x[i];
        bad |= c > lim || c < -lim;
    }
    if (__any(bad) && (threadIdx.x & 63) == 0) set_status(dev_status, ISEG_DEV_RANGE);
}
}  // namespace

bool prof_claim(int kid, hipEvent_t* start, hipEvent_t* stop)
{
    if (kid == ISEG_KID_NONE || g_kid.load(std::memory_order_relaxed) != kid) return false;
    std::lock_guard<std::mutex> lk(g_mu);
    if (g_kid.load(std::memory_order_relaxed) != kid) return false;
    g_kid.store(ISEG_KID_NONE, std::memory_order_relaxed);
    *start = g_start;
    *stop = g_stop;
    return true;
}

hipEvent_t prof_begin(int kid, hipStream_t s)
{
    hipEvent_t start, stop;
    if (!prof_claim(kid, &start, &stop)) return nullptr;
    hipEventRecord(start, s);
    return stop;
}

void prof_end(hipEvent_t stop, hipStream_t s) { hipEventRecord(stop, s); }

extern "C" int iseg_profile_arm(int32_t kernel_id, hipEvent_t start, hipEvent_t stop)
{
    if (kernel_id < ISEG_KID_NONE || kernel_id > ISEG_KID_MAXPOOL_BWD) return ISEG_ERR_ARG;
    if (kernel_id != ISEG_KID_NONE && (!start || !stop)) return ISEG_ERR_ARG;
    std::lock_guard<std::mutex> lk(g_mu);
    g_start = start;
    g_stop = stop;
    g_kid.store(kernel_id, std::memory_order_relaxed);
    return ISEG_OK;
}

void conv_plan_set(const char* name) { t_conv_plan = name; }

extern "C" const char* iseg_conv_last_plan(void) { return t_conv_plan; }

extern "C" int iseg_status_read(const int32_t* dev_status, int32_t* value, hipStream_t stream)
{
    if (!dev_status || !value) return ISEG_ERR_ARG;
    if (hipMemcpyAsync(value, dev_status, sizeof(int32_t), hipMemcpyDeviceToHost, stream) != hipSuccess)
        return ISEG_ERR_DEVICE;
    return hipStreamSynchronize(stream) == hipSuccess ? ISEG_OK : ISEG_ERR_DEVICE;
}

extern "C" int iseg_status_clear(int32_t* dev_status, hipStream_t stream)
{
    if (!dev_status) return ISEG_ERR_ARG;
    hipLaunchKernelGGL(k_status_zero, dim3(1), dim3(1), 0, stream, dev_status);
    return launch_ok();
}

extern "C" int iseg_check_codes(const int8_t* x, int64_t n, int32_t bits, int32_t* dev_status, hipStream_t stream)
{
    if (bits < 2 || bits > 8 || n < 0 || !dev_status || (n > 0 && !x)) return ISEG_ERR_ARG;
    if (((uintptr_t)x & 15) != 0) return ISEG_ERR_ARG;
    if (n == 0) return ISEG_OK;
    hipLaunchKernelGGL(k_check_codes, dim3(grid_for(n, 256 * 16, 2048)), dim3(256), 0, stream, x, n,
                       (1 << (bits - 1)) - 1, dev_status);
    return launch_ok();
}
