// calibrate.hip -- a plain HBM stream of this library's own, for roofline
// calibration only (it is no step of any operator): what one MI355X sustains
// for a copy or a read, the floors the operators' achieved bandwidth is read
// against.
//
//   stream_copy  each wave copies 64 * V consecutive 16-byte vectors (V KiB):
//                all non-temporal loads issued, then non-temporal stores;
//                V = 4 in general and V = 1 for copies of at most 8 MiB, the
//                fastest of 1 to 8 KiB per wave and 64 to 512 threads per
//                workgroup measured at 4, 16 and 256 MiB (4 MiB: 2.66 us at
//                1 KiB against 2.88 us at 4 KiB; 16 and 256 MiB: 4 KiB best).
//   stream_read  each wave reads 2 KiB (two non-temporal 16-byte loads per
//                lane) and writes one 64-bit ballot whose bit L is the parity
//                of the 32 bytes lane L read: the floor of an operator that
//                reads much and writes little, with every byte read deciding
//                the output.  Reading 12.25 MiB: 2 KiB per wave 3.55 us
//                against 3.69 us for 4 KiB; the ballot costs 0.04 us over a
//                wave that stores one lane's data unreduced, where an XOR
//                butterfly of four words over the wave through DPP moves
//                costs 0.42 us and through ds_bpermute shuffles 0.55 us,
//                each showing in the floor.
#include <stdint.h>

#include "kf_device.hpp"
#include "kf_internal.h"

namespace kf {
namespace {

constexpr int kCopyNT = 256;
constexpr int kReadVecs = 2;  // 16-byte vectors per lane in stream_read: 2 KiB per wave

template <int V>
__global__ __launch_bounds__(kCopyNT) void stream_copy(const u32x4* __restrict__ x, u32x4* __restrict__ y,
                                                       int64_t n16) {
    const int64_t wave = ((int64_t)blockIdx.x * kCopyNT + threadIdx.x) / kWave;
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t base = wave * kWave * V;
    u32x4 v[V];
#pragma unroll
    for (int k = 0; k < V; ++k) {
        const int64_t i = base + k * kWave + lane;
        v[k] = __builtin_nontemporal_load(x + (i < n16 ? i : 0));
    }
#pragma unroll
    for (int k = 0; k < V; ++k) {
        const int64_t i = base + k * kWave + lane;
        if (i < n16) __builtin_nontemporal_store(v[k], y + i);
    }
}

__global__ __launch_bounds__(kCopyNT) void stream_read(const u32x4* __restrict__ x, uint64_t* __restrict__ out,
                                                       int64_t n16) {
    const int64_t wave = ((int64_t)blockIdx.x * kCopyNT + threadIdx.x) / kWave;
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t base = wave * kWave * kReadVecs;
    u32x4 v[kReadVecs];
#pragma unroll
    for (int k = 0; k < kReadVecs; ++k) {
        const int64_t i = base + k * kWave + lane;
        v[k] = __builtin_nontemporal_load(x + (i < n16 ? i : 0));
    }
    u32x4 acc = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int k = 0; k < kReadVecs; ++k) {
        const int64_t i = base + k * kWave + lane;
        if (i < n16) acc ^= v[k];
    }
    const uint32_t folded = acc.x ^ acc.y ^ acc.z ^ acc.w;
    const uint64_t parity = __ballot(__popc(folded) & 1);
    if (lane == 0 && base < n16) out[wave] = parity;
}

}  // namespace

kf_status stream_read_launch(const void* src, int64_t bytes, void* dst, hipStream_t s) {
    const int64_t n16 = bytes / 16;
    const int64_t per_block = (int64_t)kCopyNT * kReadVecs;
    const int64_t blocks = (n16 + per_block - 1) / per_block;
    if (blocks > INT32_MAX) {
        set_error("stream_read: %lld bytes exceed the grid limit", (long long)bytes);
        return KF_ERR_BAD_SHAPE;
    }
    hipLaunchKernelGGL(stream_read, dim3((unsigned)blocks), dim3(kCopyNT), 0, s, static_cast<const u32x4*>(src),
                       static_cast<uint64_t*>(dst), n16);
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) {
        set_error("stream_read launch failed: %s", hipGetErrorString(err));
        return KF_ERR_HIP;
    }
    return KF_OK;
}

kf_status stream_copy_launch(const void* src, void* dst, int64_t bytes, hipStream_t s) {
    const int64_t n16 = bytes / 16;
    const bool small = bytes <= ((int64_t)8 << 20);
    const int64_t per_block = (int64_t)kCopyNT * (small ? 1 : 4);
    const int64_t blocks = (n16 + per_block - 1) / per_block;
    if (blocks > INT32_MAX) {
        set_error("stream_copy: %lld bytes exceed the grid limit", (long long)bytes);
        return KF_ERR_BAD_SHAPE;
    }
    const u32x4* x = static_cast<const u32x4*>(src);
    u32x4* y = static_cast<u32x4*>(dst);
    if (small) hipLaunchKernelGGL(stream_copy<1>, dim3((unsigned)blocks), dim3(kCopyNT), 0, s, x, y, n16);
    else hipLaunchKernelGGL(stream_copy<4>, dim3((unsigned)blocks), dim3(kCopyNT), 0, s, x, y, n16);
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) {
        set_error("stream_copy launch failed: %s", hipGetErrorString(err));
        return KF_ERR_HIP;
    }
    return KF_OK;
}

}  // namespace kf
