// hip_host_stub.cpp -- host-memory stand-in for the HIP runtime calls of echo_host.cpp.
//
// TEST INFRASTRUCTURE for the sanitizer build of the loader: echo_host.cpp is
// compiled with g++ -fsanitize=address,undefined and linked against this file
// instead of the HIP runtime and the device kernels, so that validation,
// matching, levelling, walk-list construction, the upload and the walk-chain
// analysis all run on the CPU under AddressSanitizer and UBSan.  "Device"
// memory is host memory; kernel launches are refused.  Two controls for the
// tests: fail the (k+1)-th allocation from now on (forced ECHO_ERR_NOMEM), and
// count the allocations still live (nothing may leak on any error path).
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <set>

#include "echo_internal.h"

namespace {
std::mutex g_mu;
std::set<void *> g_live;
int64_t g_fail_after = -1;   // allocations left before the next one fails (-1: never)
}  // namespace

extern "C" {

void echo_stub_fail_after(int64_t k) {
    std::lock_guard<std::mutex> lk(g_mu);
    g_fail_after = k;
}

int64_t echo_stub_live_allocations(void) {
    std::lock_guard<std::mutex> lk(g_mu);
    return (int64_t)g_live.size();
}

hipError_t hipSetDevice(int) { return hipSuccess; }
hipError_t hipDeviceSynchronize(void) { return hipSuccess; }
hipError_t hipStreamSynchronize(hipStream_t) { return hipSuccess; }

hipError_t hipMalloc(void **p, size_t n) {
    std::lock_guard<std::mutex> lk(g_mu);
    *p = nullptr;
    if (g_fail_after == 0) return hipErrorOutOfMemory;
    if (g_fail_after > 0) --g_fail_after;
    *p = std::malloc(n ? n : 1);
    if (!*p) return hipErrorOutOfMemory;
    g_live.insert(*p);
    return hipSuccess;
}

hipError_t hipFree(void *p) {
    if (!p) return hipSuccess;
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_live.erase(p)) return hipErrorInvalidValue;
    std::free(p);
    return hipSuccess;
}

hipError_t hipMemcpy(void *dst, const void *src, size_t n, hipMemcpyKind) {
    if (n) std::memcpy(dst, src, n);
    return hipSuccess;
}

const char *hipGetErrorString(hipError_t e) {
    return e == hipSuccess ? "no error" : e == hipErrorOutOfMemory ? "out of memory (stub)" : "error (stub)";
}

hipError_t hipEventCreate(hipEvent_t *) { return hipErrorNotSupported; }
hipError_t hipEventDestroy(hipEvent_t) { return hipSuccess; }
hipError_t hipEventRecord(hipEvent_t, hipStream_t) { return hipErrorNotSupported; }
hipError_t hipEventElapsedTime(float *, hipEvent_t, hipEvent_t) { return hipErrorNotSupported; }

}  // extern "C"

namespace echo {

// Two eight-wavefront workgroups per compute unit on 256 compute units, for every variant.
hipError_t walk_capacity(int, int64_t workgroups[kWalkVariants]) {
    for (int v = 0; v < kWalkVariants; ++v) workgroups[v] = 512;
    return hipSuccess;
}

hipError_t launch_init(const DeviceGraph &, const echo_scenario *, int32_t, unsigned long long *, int64_t, unsigned *,
                       int64_t, int64_t *, int64_t, int64_t *, uint64_t *, hipStream_t) {
    return hipErrorNotSupported;
}
hipError_t launch_clear(unsigned long long *, int64_t, unsigned *, int64_t, int64_t *, int64_t, hipStream_t) {
    return hipErrorNotSupported;
}
hipError_t launch_cc_cost(const CollTable &, const echo_cc_table *, const echo_scenario *, int32_t, int64_t *,
                          unsigned *, hipStream_t) {
    return hipErrorNotSupported;
}
hipError_t launch_walk(const WalkArgs &, int32_t, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_overlap(const OverlapArgs &, int32_t, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_settle(unsigned *, int32_t, int32_t *, unsigned *, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_fill_i32(int32_t *, int64_t, int32_t, hipStream_t) { return hipErrorNotSupported; }
// the bins stay unset on the CPU: no compose runs there
hipError_t launch_forest_bins(const DeviceGraph &, int64_t, const CompactForest &, hipStream_t) { return hipSuccess; }
hipError_t scratch_buffer(int, void **ptr) {
    *ptr = nullptr;
    return hipErrorNotSupported;
}

}  // namespace echo
