// Per-device launch facts that never change once known: the dynamic-LDS limit
// set on each kernel that needs more than the default, and the resident
// workgroups per CU of the persistent kernels.  Querying or setting them costs
// several microseconds of host time per runtime call, more than some of the
// launches they serve, so each is done once per device and kernel.
#include <hip/hip_runtime.h>

#include <mutex>

#include "kernels.hpp"

namespace isam {
namespace {

constexpr int kDevs = 64, kEntries = 128;

struct LdsEntry {
    const void* fn;
    size_t lds;
};
struct OccEntry {
    const void* fn;
    int threads;
    size_t lds;
    int value;
};

std::mutex g_mu;
LdsEntry g_lds[kDevs][kEntries];
OccEntry g_occ[kDevs][kEntries];

int current_device() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kDevs) {
        (void)hipGetLastError();
        return -1;
    }
    return dev;
}

}  // namespace

hipError_t ensure_dynamic_lds(const void* fn, size_t lds) {
    const int dev = current_device();
    std::unique_lock<std::mutex> lk(g_mu, std::defer_lock);
    try {
        lk.lock();
    } catch (...) {
        return hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    }
    LdsEntry* slot = nullptr;
    if (dev >= 0) {
        for (LdsEntry& e : g_lds[dev]) {
            if (e.fn == fn) {
                if (e.lds >= lds) return hipSuccess;
                slot = &e;
                break;
            }
            if (!e.fn) {
                slot = &e;
                break;
            }
        }
    }
    const hipError_t err = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (err == hipSuccess && slot) {
        slot->fn = fn;
        slot->lds = lds;
    }
    return err;
}

int resident_per_cu(const void* fn, int threads, size_t lds) {
    if (ensure_dynamic_lds(fn, lds) != hipSuccess) {
        (void)hipGetLastError();
        return 0;
    }
    const int dev = current_device();
    std::unique_lock<std::mutex> lk(g_mu, std::defer_lock);
    try {
        lk.lock();
    } catch (...) {
        return 0;
    }
    OccEntry* slot = nullptr;
    if (dev >= 0) {
        for (OccEntry& e : g_occ[dev]) {
            if (e.fn == fn && e.threads == threads && e.lds == lds) return e.value;
            if (!e.fn) {
                slot = &e;
                break;
            }
        }
    }
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, fn, threads, lds) != hipSuccess) {
        (void)hipGetLastError();
        return 0;
    }
    if (slot) *slot = OccEntry{fn, threads, lds, n};
    return n;
}

}  // namespace isam
