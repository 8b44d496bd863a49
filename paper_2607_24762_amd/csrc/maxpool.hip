// maxpool.hip -- max_pool2d for gfx950 (PyTorch `max_pool2d(x, kernel,
// stride, padding, dilation, ceil_mode, return_indices)` semantics), the
// max_pool2d of the paper's ResNet-50 results (Section IV-C).
//
// Max pooling selects an element; it never rounds.  Every kernel keeps the
// chosen element's raw bits and stores them, so outputs equal the input
// element bit for bit (NaN payloads included).  Selection, in row-major
// window order: start at -inf on the window's first in-plane position, move
// to any element that is greater or NaN.  Ties therefore keep the first
// position and a window holding NaN reports its last NaN; padding is never
// chosen.  Indices are row * w + col within the plane, as int64.
//
//   mp_band    NCHW.  One workgroup per (plane, band of output rows): the
//              band's input rows are one contiguous span of the plane,
//              staged into LDS with coalesced 16-byte loads; windows are
//              scanned from LDS and consecutive threads write consecutive
//              outputs.
//   mp_direct  NCHW planes whose band tile does not fit in LDS: one thread
//              per output, window loads from global memory.
//   mp_nhwc    channels last: one thread per (output pixel, 16-byte vector
//              of channels), so every window load is coalesced along C and
//              overlapping windows re-read from cache.
#include <math.h>

#include "kf_device.hpp"
#include "kf_internal.h"

namespace kf {
namespace {

constexpr int kNT = 256;
constexpr int kBandBytes = 16 << 10;  // LDS budget of one band tile

// Raw storage type of an element and its value as a float (exact).
template <class T>
struct Raw;
template <>
struct Raw<F32> {
    using type = uint32_t;
    static constexpr uint32_t neg_inf = 0xff800000u;
    __device__ static float value(uint32_t b) { return __uint_as_float(b); }
};
template <>
struct Raw<BF16> {
    using type = uint16_t;
    static constexpr uint32_t neg_inf = 0xff80u;
    __device__ static float value(uint32_t b) { return __uint_as_float(b << 16); }
};
template <>
struct Raw<F16> {
    using type = uint16_t;
    static constexpr uint32_t neg_inf = 0xfc00u;
    __device__ static float value(uint32_t b) { return (float)__builtin_bit_cast(_Float16, (uint16_t)b); }
};

// VEC raw elements as one 16-byte register value.
template <class R, int N>
struct alignas(16) Lanes {
    R v[N];
};

// The running choice of one window.
template <class T>
struct Pick {
    float best = -INFINITY;
    uint32_t bits = Raw<T>::neg_inf;
    int32_t at = -1;
    __device__ __forceinline__ void consider(uint32_t raw, int32_t pos) {
        const float v = Raw<T>::value(raw);
        if (at < 0) at = pos;
        if (v > best || v != v) {
            best = v;
            bits = raw;
            at = pos;
        }
    }
};

struct MPParams {
    const void* x;
    void* y;
    int64_t* idx;
    int64_t planes;  // NCHW: n * c
    int32_t n, c, h, w, oh, ow;
    int32_t kh, kw, sh, sw, ph, pw, dh, dw;
    int32_t band_rows, bands;  // mp_band: output rows per band, bands per plane
};

// --------------------------------------------------------------------------
// NCHW, one workgroup per (plane, band of output rows), input rows in LDS.
template <class T, bool VECTOR>
__global__ __launch_bounds__(kNT) void mp_band(MPParams p) {
    using R = typename Raw<T>::type;
    constexpr int VEC = 16 / sizeof(R);
    extern __shared__ u32x4 lds_vec[];
    R* tile = reinterpret_cast<R*>(lds_vec);
    const int64_t plane = blockIdx.x / p.bands;
    const int band = (int)(blockIdx.x - plane * p.bands);
    const int o0 = band * p.band_rows;
    const int o1 = min(p.oh, o0 + p.band_rows);
    const int r_lo = max(0, o0 * p.sh - p.ph);
    const int r_hi = min(p.h, (o1 - 1) * p.sh - p.ph + (p.kh - 1) * p.dh + 1);
    const int n = max(0, r_hi - r_lo) * p.w;
    const R* src = static_cast<const R*>(p.x) + plane * p.h * p.w + (int64_t)r_lo * p.w;

    // Stage the span; in the vector form every band starts on a 16-byte
    // boundary (w and h*w are whole vectors, the base is aligned) and the
    // span is whole vectors.  Four loads in flight per thread.
    if constexpr (VECTOR) {
        const u32x4* s4 = reinterpret_cast<const u32x4*>(src);
        const int nv = n / VEC;
        for (int v0 = threadIdx.x; v0 < nv; v0 += 4 * kNT) {
            u32x4 r[4];
#pragma unroll
            for (int d = 0; d < 4; ++d) {
                const int v = v0 + d * kNT;
                r[d] = s4[v < nv ? v : 0];
            }
#pragma unroll
            for (int d = 0; d < 4; ++d)
                if (v0 + d * kNT < nv) lds_vec[v0 + d * kNT] = r[d];
        }
    } else {
        for (int e = threadIdx.x; e < n; e += kNT) tile[e] = src[e];
    }
    __syncthreads();

    const int outs = (o1 - o0) * p.ow;
    R* dst = static_cast<R*>(p.y) + plane * p.oh * p.ow + (int64_t)o0 * p.ow;
    for (int q = threadIdx.x; q < outs; q += kNT) {
        const int i = o0 + q / p.ow, j = q - (q / p.ow) * p.ow;
        Pick<T> pk;
        for (int a = 0; a < p.kh; ++a) {
            const int r = i * p.sh - p.ph + a * p.dh;
            if (r < 0 || r >= p.h) continue;
            const R* row = tile + (r - r_lo) * p.w;
            for (int b = 0; b < p.kw; ++b) {
                const int col = j * p.sw - p.pw + b * p.dw;
                if (col < 0 || col >= p.w) continue;
                pk.consider(row[col], r * p.w + col);
            }
        }
        dst[q] = (R)pk.bits;
        if (p.idx) p.idx[plane * p.oh * p.ow + (int64_t)o0 * p.ow + q] = pk.at;
    }
}

// --------------------------------------------------------------------------
// NCHW fallback: one thread per output, window loads from global memory.
template <class T>
__global__ __launch_bounds__(kNT) void mp_direct(MPParams p) {
    using R = typename Raw<T>::type;
    const int64_t o = (int64_t)blockIdx.x * kNT + threadIdx.x;
    const int64_t per_plane = (int64_t)p.oh * p.ow;
    if (o >= p.planes * per_plane) return;
    const int64_t plane = o / per_plane;
    const int q = (int)(o - plane * per_plane);
    const int i = q / p.ow, j = q - (q / p.ow) * p.ow;
    const R* xp = static_cast<const R*>(p.x) + plane * p.h * p.w;
    Pick<T> pk;
    for (int a = 0; a < p.kh; ++a) {
        const int r = i * p.sh - p.ph + a * p.dh;
        if (r < 0 || r >= p.h) continue;
        for (int b = 0; b < p.kw; ++b) {
            const int col = j * p.sw - p.pw + b * p.dw;
            if (col < 0 || col >= p.w) continue;
            pk.consider(xp[(int64_t)r * p.w + col], r * p.w + col);
        }
    }
    static_cast<R*>(p.y)[o] = (R)pk.bits;
    if (p.idx) p.idx[o] = pk.at;
}

// --------------------------------------------------------------------------
// NHWC: thread per (output pixel, VEC channels).  VEC = 16 bytes of
// channels when c is whole vectors and the bases are aligned, else 1.
template <class T, int VEC>
__global__ __launch_bounds__(kNT) void mp_nhwc(MPParams p) {
    using R = typename Raw<T>::type;
    const int cvs = p.c / VEC;
    const int64_t t = (int64_t)blockIdx.x * kNT + threadIdx.x;
    const int64_t total = (int64_t)p.n * p.oh * p.ow * cvs;
    if (t >= total) return;
    const int cv = (int)(t % cvs);
    const int64_t pix = t / cvs;
    const int j = (int)(pix % p.ow);
    const int i = (int)((pix / p.ow) % p.oh);
    const int64_t nn = pix / ((int64_t)p.ow * p.oh);
    const R* xs = static_cast<const R*>(p.x);
    Pick<T> pk[VEC];
    for (int a = 0; a < p.kh; ++a) {
        const int r = i * p.sh - p.ph + a * p.dh;
        if (r < 0 || r >= p.h) continue;
        for (int b = 0; b < p.kw; ++b) {
            const int col = j * p.sw - p.pw + b * p.dw;
            if (col < 0 || col >= p.w) continue;
            const int64_t e = ((nn * p.h + r) * p.w + col) * p.c + (int64_t)cv * VEC;
            Lanes<R, VEC> v;
            if constexpr (VEC == 1) {
                v.v[0] = xs[e];
            } else {
                v = __builtin_bit_cast(Lanes<R, VEC>, *reinterpret_cast<const u32x4*>(xs + e));
            }
#pragma unroll
            for (int k = 0; k < VEC; ++k) pk[k].consider(v.v[k], r * p.w + col);
        }
    }
    const int64_t o = pix * p.c + (int64_t)cv * VEC;
    Lanes<R, VEC> out;
#pragma unroll
    for (int k = 0; k < VEC; ++k) out.v[k] = (R)pk[k].bits;
    if constexpr (VEC == 1) {
        static_cast<R*>(p.y)[o] = out.v[0];
    } else {
        *reinterpret_cast<u32x4*>(static_cast<R*>(p.y) + o) = __builtin_bit_cast(u32x4, out);
    }
    if (p.idx) {
#pragma unroll
        for (int k = 0; k < VEC; ++k) p.idx[o + k] = pk[k].at;
    }
}

// --------------------------------------------------------------------------
// Host side.
template <class T>
kf_status run(const MaxPoolArgs& a, hipStream_t s, const char** variant) {
    using R = typename Raw<T>::type;
    constexpr int VEC = 16 / sizeof(R);
    MPParams p;
    p.x = a.x;
    p.y = a.y;
    p.idx = a.idx;
    p.planes = a.n * a.c;
    p.n = (int32_t)a.n;
    p.c = (int32_t)a.c;
    p.h = (int32_t)a.h;
    p.w = (int32_t)a.w;
    p.oh = (int32_t)a.oh;
    p.ow = (int32_t)a.ow;
    p.kh = a.kh;
    p.kw = a.kw;
    p.sh = a.sh;
    p.sw = a.sw;
    p.ph = a.ph;
    p.pw = a.pw;
    p.dh = a.dh;
    p.dw = a.dw;
    p.band_rows = p.bands = 1;
    if (a.nhwc) {
        const bool vec = a.c % VEC == 0 && (uintptr_t)a.x % 16 == 0 && (uintptr_t)a.y % 16 == 0;
        const int64_t threads = a.n * a.oh * a.ow * (vec ? a.c / VEC : a.c);
        const int64_t blocks = (threads + kNT - 1) / kNT;
        if (blocks > INT32_MAX) {
            set_error("max_pool2d: grid of %lld workgroups exceeds the launch limit", (long long)blocks);
            return KF_ERR_UNSUPPORTED_LAYOUT;
        }
        if (vec) {
            hipLaunchKernelGGL((mp_nhwc<T, VEC>), dim3((unsigned)blocks), dim3(kNT), 0, s, p);
            *variant = "mp_nhwc_vec";
        } else {
            hipLaunchKernelGGL((mp_nhwc<T, 1>), dim3((unsigned)blocks), dim3(kNT), 0, s, p);
            *variant = "mp_nhwc_scalar";
        }
    } else {
        // Output rows per band: as many as keep the band's input rows within
        // kBandBytes, then evened out over the plane's bands.
        const int64_t row_bytes = a.w * (int64_t)sizeof(R);
        const int64_t max_in_rows = kBandBytes / row_bytes;
        const int64_t eff = (int64_t)(a.kh - 1) * a.dh + 1;  // input rows one window spans
        int64_t br = max_in_rows >= eff ? (max_in_rows - eff) / a.sh + 1 : 0;
        if (br >= 1) {
            br = br < a.oh ? br : a.oh;
            const int64_t bands = (a.oh + br - 1) / br;
            br = (a.oh + bands - 1) / bands;
            p.band_rows = (int32_t)br;
            p.bands = (int32_t)bands;
            const int64_t grid = p.planes * bands;
            if (grid > INT32_MAX) {
                set_error("max_pool2d: grid of %lld workgroups exceeds the launch limit", (long long)grid);
                return KF_ERR_UNSUPPORTED_LAYOUT;
            }
            const int64_t in_rows = (br - 1) * a.sh + eff;
            const size_t lds = (size_t)(((in_rows * row_bytes) + 15) / 16 * 16);
            const bool vec = a.w % VEC == 0 && (a.h * a.w) % VEC == 0 && (uintptr_t)a.x % 16 == 0;
            if (vec) {
                hipLaunchKernelGGL((mp_band<T, true>), dim3((unsigned)grid), dim3(kNT), lds, s, p);
                *variant = "mp_band_vec";
            } else {
                hipLaunchKernelGGL((mp_band<T, false>), dim3((unsigned)grid), dim3(kNT), lds, s, p);
                *variant = "mp_band_scalar";
            }
        } else {
            const int64_t blocks = (p.planes * a.oh * a.ow + kNT - 1) / kNT;
            if (blocks > INT32_MAX) {
                set_error("max_pool2d: grid of %lld workgroups exceeds the launch limit", (long long)blocks);
                return KF_ERR_UNSUPPORTED_LAYOUT;
            }
            hipLaunchKernelGGL((mp_direct<T>), dim3((unsigned)blocks), dim3(kNT), 0, s, p);
            *variant = "mp_direct";
        }
    }
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) {
        set_error("max_pool2d launch failed: %s", hipGetErrorString(err));
        return KF_ERR_HIP;
    }
    return KF_OK;
}

}  // namespace

kf_status max_pool2d_launch(const MaxPoolArgs& a, hipStream_t s, const char** variant) {
    switch (a.t) {
        case KF_FLOAT32: return run<F32>(a, s, variant);
        case KF_BFLOAT16: return run<BF16>(a, s, variant);
        case KF_FLOAT16: return run<F16>(a, s, variant);
    }
    set_error("max_pool2d: unsupported dtype");
    return KF_ERR_BAD_DTYPE;
}

}  // namespace kf
