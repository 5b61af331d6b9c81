// launch.hip -- host-side launch helpers shared by the kernel files.
#include <mutex>
#include <unordered_map>

#include "iseg_common.h"

namespace {
struct KeyHash {
    size_t operator()(const std::pair<int, const void*>& k) const
    {
        return std::hash<const void*>()(k.second) ^ ((size_t)k.first << 48);
    }
};
std::mutex g_lds_mu;
std::unordered_map<std::pair<int, const void*>, int, KeyHash> g_lds_set;   // (device, kernel) -> bytes
}  // namespace

// Raise a kernel's dynamic LDS limit to at least `bytes` on the current
// device.  The attribute call costs host time, so each (device, kernel) pair
// makes it only when a launch needs more than it has already been given.
bool lds_limit(const void* f, size_t bytes)
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return false;
    const std::pair<int, const void*> key(dev, f);
    std::lock_guard<std::mutex> lock(g_lds_mu);
    auto it = g_lds_set.find(key);
    if (it != g_lds_set.end() && (size_t)it->second >= bytes) return true;
    if (hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes) != hipSuccess) return false;
    g_lds_set[key] = (int)bytes;
    return true;
}
