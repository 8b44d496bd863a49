// runtime.cpp -- per-device properties the launch code needs, queried once
// per device and cached, and the environment knobs read once per process.
#include <atomic>
#include <cstdlib>

#include "kf_internal.h"

namespace kf {

namespace {
constexpr int kMaxDevices = 64;

// value + 1 in an atomic, 0 meaning not yet known.
int cached_attr(std::atomic<int>* cache, int dev, hipDeviceAttribute_t attr) {
    if (dev < 0 || dev >= kMaxDevices) return 0;
    int v = cache[dev].load(std::memory_order_relaxed);
    if (v == 0) {
        int got = 0;
        if (hipDeviceGetAttribute(&got, attr, dev) != hipSuccess) got = 0;
        v = got + 1;
        cache[dev].store(v, std::memory_order_relaxed);
    }
    return v - 1;
}
}  // namespace

int device_multiprocessors(int dev) {
    static std::atomic<int> cache[kMaxDevices];
    return cached_attr(cache, dev, hipDeviceAttributeMultiprocessorCount);
}

bool device_cooperative(int dev) {
    static std::atomic<int> cache[kMaxDevices];
    return cached_attr(cache, dev, hipDeviceAttributeCooperativeLaunch) != 0;
}

int resident_capacity(ResidencyCache& cache, int dev, const void* kernel, int threads) {
    if (dev < 0 || dev >= ResidencyCache::kDevices) return 0;
    int v = cache.v[dev].load(std::memory_order_relaxed);
    if (v == 0) {
        int per_cu = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, 0) != hipSuccess) per_cu = 0;
        v = per_cu * device_multiprocessors(dev) + 1;
        cache.v[dev].store(v, std::memory_order_relaxed);
    }
    return v - 1;
}

uint32_t env_u32(const char* name, uint32_t dflt) {
    const char* e = std::getenv(name);
    return e ? (uint32_t)std::strtoul(e, nullptr, 10) : dflt;
}

}  // namespace kf
