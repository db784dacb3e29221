// Host-side caches shared by the entry points: kernel LDS attributes, each
// kernel's static LDS and the compute-unit count of each device, each looked
// up once per process.
#include <mutex>
#include <unordered_map>

#include "maps_internal.hpp"

namespace maps {

void allow_dynamic_lds_fn(const void* fn, size_t bytes) {
    static std::mutex mu;
    static std::unordered_map<const void*, size_t> done;
    std::lock_guard<std::mutex> lock(mu);
    auto it = done.find(fn);
    if (it != done.end() && it->second >= bytes) return;
    (void)hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, int(bytes));
    (void)hipGetLastError();   // a refused attribute shows up at the launch instead
    done[fn] = bytes;
}

int device_compute_units() {
    static std::mutex mu;
    static std::unordered_map<int, int> cus;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 256;
    std::lock_guard<std::mutex> lock(mu);
    auto it = cus.find(dev);
    if (it != cus.end()) return it->second;
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) v = 256;
    cus[dev] = v;
    return v;
}

size_t kernel_static_lds(const void* fn) {
    static std::mutex mu;
    static std::unordered_map<const void*, size_t> sizes;
    std::lock_guard<std::mutex> lock(mu);
    auto it = sizes.find(fn);
    if (it != sizes.end()) return it->second;
    hipFuncAttributes fa{};
    // unknown: assume the whole workgroup's LDS is taken, so that no dynamic LDS is planned
    const size_t v = hipFuncGetAttributes(&fa, fn) == hipSuccess ? fa.sharedSizeBytes : kLdsPerWorkgroup;
    (void)hipGetLastError();
    sizes[fn] = v;
    return v;
}

}  // namespace maps
