// profile.hip -- the in-place kernel timing hook (iseg_profile_arm).
#include "iseg_common.h"

namespace {
int g_kid = ISEG_KID_NONE;
hipEvent_t g_start = nullptr, g_stop = nullptr;
}  // namespace

bool prof_begin(int kid, hipStream_t s)
{
    if (g_kid != kid || kid == ISEG_KID_NONE) return false;
    hipEventRecord(g_start, s);
    return true;
}

void prof_end(int kid, hipStream_t s)
{
    (void)kid;
    hipEventRecord(g_stop, s);
    g_kid = ISEG_KID_NONE;
}

extern "C" int iseg_profile_arm(int32_t kernel_id, hipEvent_t start, hipEvent_t stop)
{
    if (kernel_id < ISEG_KID_NONE || kernel_id > ISEG_KID_MAXPOOL_BWD) return ISEG_ERR_ARG;
    if (kernel_id != ISEG_KID_NONE && (!start || !stop)) return ISEG_ERR_ARG;
    g_kid = kernel_id;
    g_start = start;
    g_stop = stop;
    return ISEG_OK;
}
