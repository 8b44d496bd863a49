// calibrate.hip -- a plain HBM stream of this library's own, for roofline
// calibration only (it is no step of any operator): what one MI355X sustains
// for a copy, the figure the operators' achieved bandwidth is read against.
//
//   stream_copy  each wave copies 64 * kCopyVecs consecutive 16-byte vectors
//                (4 KiB): all non-temporal loads issued, then non-temporal
//                stores, the pattern that measured fastest among grid-strided
//                and wave-contiguous copies with 1-16 vectors per lane and
//                among the cache-policy bits of loads and stores.
//   stream_read  the same loads; each wave writes only the XOR of its 4 KiB
//                (one 16-byte word), so the bytes moved are the read: the
//                floor of an operator that reads much and writes little.
#include <stdint.h>

#include "kf_device.hpp"
#include "kf_internal.h"

namespace kf {
namespace {

constexpr int kCopyNT = 256;
constexpr int kCopyVecs = 4;  // 16-byte vectors per lane: 4 KiB per wave

__global__ __launch_bounds__(kCopyNT) void stream_copy(const u32x4* __restrict__ x, u32x4* __restrict__ y,
                                                       int64_t n16) {
    const int64_t wave = ((int64_t)blockIdx.x * kCopyNT + threadIdx.x) / kWave;
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t base = wave * kWave * kCopyVecs;
    u32x4 v[kCopyVecs];
#pragma unroll
    for (int k = 0; k < kCopyVecs; ++k) {
        const int64_t i = base + k * kWave + lane;
        v[k] = __builtin_nontemporal_load(x + (i < n16 ? i : 0));
    }
#pragma unroll
    for (int k = 0; k < kCopyVecs; ++k) {
        const int64_t i = base + k * kWave + lane;
        if (i < n16) __builtin_nontemporal_store(v[k], y + i);
    }
}

__global__ __launch_bounds__(kCopyNT) void stream_read(const u32x4* __restrict__ x, u32x4* __restrict__ out,
                                                       int64_t n16) {
    const int64_t wave = ((int64_t)blockIdx.x * kCopyNT + threadIdx.x) / kWave;
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t base = wave * kWave * kCopyVecs;
    u32x4 v[kCopyVecs];
#pragma unroll
    for (int k = 0; k < kCopyVecs; ++k) {
        const int64_t i = base + k * kWave + lane;
        v[k] = __builtin_nontemporal_load(x + (i < n16 ? i : 0));
    }
    u32x4 acc = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int k = 0; k < kCopyVecs; ++k) {
        const int64_t i = base + k * kWave + lane;
        if (i < n16) acc ^= v[k];
    }
#pragma unroll
    for (int o = kWave / 2; o >= 1; o >>= 1) {
#pragma unroll
        for (int w = 0; w < 4; ++w) acc[w] ^= (uint32_t)__shfl_xor((int)acc[w], o);
    }
    if (lane == 0 && base < n16) __builtin_nontemporal_store(acc, out + wave);
}

}  // namespace

kf_status stream_read_launch(const void* src, int64_t bytes, void* dst, hipStream_t s) {
    const int64_t n16 = bytes / 16;
    const int64_t per_block = (int64_t)kCopyNT * kCopyVecs;
    const int64_t blocks = (n16 + per_block - 1) / per_block;
    if (blocks > INT32_MAX) {
        set_error("stream_read: %lld bytes exceed the grid limit", (long long)bytes);
        return KF_ERR_BAD_SHAPE;
    }
    hipLaunchKernelGGL(stream_read, dim3((unsigned)blocks), dim3(kCopyNT), 0, s, static_cast<const u32x4*>(src),
                       static_cast<u32x4*>(dst), n16);
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) {
        set_error("stream_read launch failed: %s", hipGetErrorString(err));
        return KF_ERR_HIP;
    }
    return KF_OK;
}

kf_status stream_copy_launch(const void* src, void* dst, int64_t bytes, hipStream_t s) {
    const int64_t n16 = bytes / 16;
    const int64_t per_block = (int64_t)kCopyNT * kCopyVecs;
    const int64_t blocks = (n16 + per_block - 1) / per_block;
    if (blocks > INT32_MAX) {
        set_error("stream_copy: %lld bytes exceed the grid limit", (long long)bytes);
        return KF_ERR_BAD_SHAPE;
    }
    hipLaunchKernelGGL(stream_copy, dim3((unsigned)blocks), dim3(kCopyNT), 0, s, static_cast<const u32x4*>(src),
                       static_cast<u32x4*>(dst), n16);
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) {
        set_error("stream_copy launch failed: %s", hipGetErrorString(err));
        return KF_ERR_HIP;
    }
    return KF_OK;
}

}  // namespace kf
