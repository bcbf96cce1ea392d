// Allocation-free dense evaluation: dss_eval_dense with its workspace in a
// fixed device array of the library instead of a caller or plan buffer, for
// callers that cannot allocate device memory.
//
// The array is a file-scope device variable.  Its name, used in host code, is
// a host-side stand-in and not a device address; the device address is looked
// up with hipGetSymbolAddress once per device, on the entry point's first call
// with that device current, and kept in a per-device table.  Only that address
// is ever handed to a kernel.  Every call on one device shares that device's
// array: calls that overlap on a device (several streams or host threads) race.
// Nothing in it has to start at zero: every kernel of the dense evaluation
// writes each workspace byte it reads earlier in the same evaluation.
#include <mutex>
#include <vector>

#include "dss_internal.h"

// 64 MiB: the ping-pong intermediates of signals of up to about 10^5 samples
// at the named workloads' channel widths (the 64x64 workload needs 0.19 MB, a
// 200x200 signal through the 512x512 workload's network 38 MB, 10^5 samples
// through the 1-D network 51 MB).
static constexpr int64_t kScratchBytes = DSS_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) char scratch[kScratchBytes];

namespace {

std::mutex g_scratch_mu;
std::vector<char*> g_scratch_ptr;   // per device: the device address of `scratch`, or nullptr

// The device address of the scratch array on the current device `dev`.
dss_status scratch_address(int dev, char** ptr) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if ((int)g_scratch_ptr.size() <= dev) g_scratch_ptr.resize(dev + 1, nullptr);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return dss::hip_fail(e, "hipGetSymbolAddress of the scratch array");
        if (!p || ((uintptr_t)p & 255u) != 0) return dss::fail(DSS_E_HIP, "scratch array at an unaligned address");
        g_scratch_ptr[dev] = static_cast<char*>(p);
    }
    *ptr = g_scratch_ptr[dev];
    return DSS_OK;
}

}  // namespace

extern "C" dss_status dss_eval_dense_noalloc(dss_plan_t plan, const void* signal, int32_t H, int32_t W, float* out,
                                             hipStream_t stream) {
    dss::Geom G;
    dss_status s = dss::eval_prepare(plan, signal, out, H, W, 0, &G);
    if (s != DSS_OK) return s;
    if (G.ws_bytes > kScratchBytes)
        return dss::fail(DSS_E_UNSUPPORTED,
                         "a %dx%d signal needs %lld bytes of workspace; the allocation-free evaluation has %lld",
                         H, W, (long long)G.ws_bytes, (long long)kScratchBytes);
    char* ws = nullptr;
    s = scratch_address(plan->device, &ws);
    if (s != DSS_OK) return s;
    return dss::eval_run(plan, G, signal, out, ws, stream, false);
}
