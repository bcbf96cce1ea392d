// Device attributes the kernel launchers need: the largest dynamic LDS
// allocation of a workgroup, and the per-kernel opt-in above 64 KB.  Both are
// kept per device (a kernel attribute is set for the current device) and may be
// called from several host threads at once.
#include <mutex>
#include <vector>

#include "dss_internal.h"

namespace dss {

namespace {
std::mutex g_mu;
struct LdsLimit {
    int dev;
    int bytes;
};
struct LdsOptIn {
    int dev;
    const void* kern;
    size_t bytes;
};
std::vector<LdsLimit> g_limits;
std::vector<LdsOptIn> g_opt_ins;
}  // namespace

size_t device_lds_limit() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 64 * 1024;
    std::lock_guard<std::mutex> lock(g_mu);
    for (const LdsLimit& l : g_limits)
        if (l.dev == dev) return (size_t)l.bytes;
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess) v = 64 * 1024;
    g_limits.push_back({dev, v});
    return (size_t)v;
}

hipError_t allow_dynamic_lds(const void* kern, size_t bytes) {
    if (bytes <= 64 * 1024) return hipSuccess;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    std::lock_guard<std::mutex> lock(g_mu);
    LdsOptIn* known = nullptr;
    for (LdsOptIn& o : g_opt_ins)
        if (o.dev == dev && o.kern == kern) known = &o;
    if (known && known->bytes >= bytes) return hipSuccess;
    e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    if (e != hipSuccess) return e;
    if (known)
        known->bytes = bytes;
    else
        g_opt_ins.push_back({dev, kern, bytes});
    return hipSuccess;
}

}  // namespace dss
