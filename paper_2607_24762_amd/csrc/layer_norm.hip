// layer_norm.hip -- LayerNorm for gfx950 (PyTorch `layer_norm(x,
// normalized_shape, w, b, eps)` semantics: per row of the d trailing
// elements, biased variance, eps inside the square root, elementwise
// affine), the operator of the paper's SD3.5 Medium layer_norm result
// (Section IV-C).
//
//   ln_wave   LPR lanes own a row held in registers (64/LPR rows per wave);
//             moments merge by a butterfly inside the lane group.
//   ln_block  one workgroup per row held in registers, each wave streaming a
//             contiguous stretch; per-wave moments merge through LDS.
//   ln_stream one workgroup per row of any length: a moments pass, then a
//             normalise pass that reads the row again.
//
// Per-thread moments use sums shifted by the mean of the thread's first
// 16-byte slot (folded in as loads land), converted to (count, mean, M2) and
// combined with the Chan update (kf_device.hpp).  Loads are unconditional
// (out-of-range slots re-read the row's first element and are excluded from
// the sums); stores are non-temporal.
#include <math.h>

#include <type_traits>

#include "kf_device.hpp"
#include "kf_internal.h"

namespace kf {
namespace {

// VEC consecutive affine values (type A) starting at element e: 16-byte
// loads when VECTOR (the caller guarantees alignment), else one at a time.
template <class A, int VEC, bool VECTOR>
__device__ __forceinline__ void load_affine_span(const void* p, int64_t e, float* out) {
    if constexpr (VECTOR) {
#pragma unroll
        for (int i = 0; i < VEC / A::vec; ++i) load_vec<A>(p, e + i * A::vec, out + i * A::vec);
    } else {
#pragma unroll
        for (int i = 0; i < VEC; ++i) out[i] = load1<A>(p, e + i);
    }
}

// Affine type of a call with neither weight nor bias: the kernels then hold
// no affine registers (no 16-byte weight / bias slots per element), which
// raises occupancy.
struct NoAffine {};

struct LNArgsDev {
    const void* x;
    void* y;
    const void* w;
    const void* b;
    int64_t rows;
    int32_t d;
    float eps;
};

// Thread moments of NV slots of VEC values, slot k valid when ok[k].
template <int NV, int VEC>
__device__ __forceinline__ Moments slot_moments(const float (&v)[NV][VEC], const bool (&ok)[NV]) {
    float K = v[0][0];
#pragma unroll
    for (int i = 1; i < VEC; ++i) K += v[0][i];
    K *= 1.f / (float)VEC;
    float s1 = 0.f, s2 = 0.f, cnt = 0.f;
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        if (ok[k]) {
            cnt += (float)VEC;
#pragma unroll
            for (int i = 0; i < VEC; ++i) {
                const float dv = v[k][i] - K;
                s1 += dv;
                s2 = fmaf(dv, dv, s2);
            }
        }
    }
    if (cnt == 0.f) return Moments{0.f, 0.f, 0.f};
    const float r = __builtin_amdgcn_rcpf(cnt);
    const float d1 = s1 * r;
    return Moments{cnt, K + d1, fmaxf(fmaf(-s1, d1, s2), 0.f)};
}

// y = (x - mean) * rstd * w[j] + b[j] for the valid slots, with
// rstd = 1 / sqrt(M2/d + eps), stored non-temporally.  Slot k starts at
// element e0[k] of the row.  16-bit outputs evaluate it in fp32; fp32
// outputs in double, rounded once (x - mean is exact there and rstd * w[j]
// carries no fp32 rounding: the output's error is one fp32 rounding plus
// what the fp32 statistics carry).
template <class T, class A, int NV, int VEC, bool VECTOR>
__device__ __forceinline__ void normalise_slots(const LNArgsDev& p, int64_t base, const int (&e0)[NV],
                                                const bool (&ok)[NV], float (&v)[NV][VEC], float mean,
                                                float m2) {
    using Acc = std::conditional_t<std::is_same_v<T, F32>, double, float>;
    Acc rstd;
    if constexpr (std::is_same_v<Acc, double>) rstd = 1.0 / sqrt((double)m2 / (double)p.d + (double)p.eps);
    else rstd = 1.f / sqrtf(m2 / (float)p.d + p.eps);
    const Acc mu = (Acc)mean;
    if constexpr (std::is_same_v<A, NoAffine>) {
#pragma unroll
        for (int k = 0; k < NV; ++k) {
            if (ok[k]) {
#pragma unroll
                for (int i = 0; i < VEC; ++i) v[k][i] = (float)(((Acc)v[k][i] - mu) * rstd);
                if constexpr (VECTOR) store_vec<T, true>(p.y, base + e0[k], v[k]);
                else store1<T>(p.y, base + e0[k], v[k][0]);
            }
        }
    } else {
        float wv[NV][VEC], bv[NV][VEC];
        if (p.w) {
#pragma unroll
            for (int k = 0; k < NV; ++k) load_affine_span<A, VEC, VECTOR>(p.w, ok[k] ? e0[k] : 0, wv[k]);
        }
        if (p.b) {
#pragma unroll
            for (int k = 0; k < NV; ++k) load_affine_span<A, VEC, VECTOR>(p.b, ok[k] ? e0[k] : 0, bv[k]);
        }
#pragma unroll
        for (int k = 0; k < NV; ++k) {
            if (ok[k]) {
#pragma unroll
                for (int i = 0; i < VEC; ++i) {
                    const Acc a = p.w ? rstd * (Acc)wv[k][i] : rstd;
                    v[k][i] = (float)fma((Acc)v[k][i] - mu, a, p.b ? (Acc)bv[k][i] : (Acc)0);
                }
                if constexpr (VECTOR) store_vec<T, true>(p.y, base + e0[k], v[k]);
                else store1<T>(p.y, base + e0[k], v[k][0]);
            }
        }
    }
}

template <class T, class A, int LPR, int NV, bool VECTOR>
__global__ __launch_bounds__(256) void ln_wave(LNArgsDev p) {
    constexpr int VEC = VECTOR ? T::vec : 1;
    constexpr int RPW = kWave / LPR;
    const int lane = threadIdx.x & (kWave - 1);
    const int lr = lane & (LPR - 1);
    const int64_t row = ((int64_t)blockIdx.x * (blockDim.x / kWave) + (threadIdx.x / kWave)) * RPW + lane / LPR;
    const bool row_ok = row < p.rows;
    const int64_t base = (row_ok ? row : 0) * (int64_t)p.d;

    float v[NV][VEC];
    int e0[NV];
    bool ok[NV];
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        e0[k] = (lr + k * LPR) * VEC;
        ok[k] = row_ok && e0[k] < p.d;
        const int64_t at = base + (ok[k] ? e0[k] : 0);
        if constexpr (VECTOR) load_vec<T, true>(p.x, at, v[k]);
        else v[k][0] = load1<T>(p.x, at);
    }
    const Moments m = moments_group<LPR>(slot_moments<NV, VEC>(v, ok));
    normalise_slots<T, A, NV, VEC, VECTOR>(p, base, e0, ok, v, m.mean, m.m2);
}

template <class T, class A, int NT, int NV, bool VECTOR>
__global__ __launch_bounds__(NT) void ln_block(LNArgsDev p) {
    constexpr int VEC = VECTOR ? T::vec : 1;
    constexpr int NW = NT / kWave;
    __shared__ Moments lds[NW];
    const int64_t base = (int64_t)blockIdx.x * p.d;
    const int lane = threadIdx.x & (kWave - 1);
    const int seg = (threadIdx.x / kWave) * NV * kWave + lane;

    float v[NV][VEC];
    int e0[NV];
    bool ok[NV];
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        e0[k] = (seg + k * kWave) * VEC;
        ok[k] = e0[k] < p.d;
        const int64_t at = base + (ok[k] ? e0[k] : 0);
        if constexpr (VECTOR) load_vec<T, true>(p.x, at, v[k]);
        else v[k][0] = load1<T>(p.x, at);
    }
    const Moments m = moments_block<NW>(slot_moments<NV, VEC>(v, ok), lds);
    normalise_slots<T, A, NV, VEC, VECTOR>(p, base, e0, ok, v, m.mean, m.m2);
}

template <class T, class A, int NT, bool VECTOR>
__global__ __launch_bounds__(NT) void ln_stream(LNArgsDev p) {
    constexpr int VEC = VECTOR ? T::vec : 1;
    constexpr int NW = NT / kWave;
    constexpr int DEPTH = 4;
    __shared__ Moments lds[NW];
    const int64_t base = (int64_t)blockIdx.x * p.d;
    // Pass 1: per-thread moments of DEPTH-slot batches, Chan-merged in order.
    Moments acc{0.f, 0.f, 0.f};
    for (int64_t e = (int64_t)threadIdx.x * VEC; e < p.d; e += (int64_t)DEPTH * NT * VEC) {
        float v[DEPTH][VEC];
        bool ok[DEPTH];
#pragma unroll
        for (int k = 0; k < DEPTH; ++k) {
            const int64_t ek = e + (int64_t)k * NT * VEC;
            ok[k] = ek < p.d;
            const int64_t at = base + (ok[k] ? ek : 0);
            if constexpr (VECTOR) load_vec<T>(p.x, at, v[k]);
            else v[k][0] = load1<T>(p.x, at);
        }
        acc = chan(acc, slot_moments<DEPTH, VEC>(v, ok));
    }
    const Moments m = moments_block<NW>(acc, lds);
    // Pass 2: normalise.
    for (int64_t e = (int64_t)threadIdx.x * VEC; e < p.d; e += (int64_t)DEPTH * NT * VEC) {
        float v[DEPTH][VEC];
        int e0[DEPTH];
        bool ok[DEPTH];
#pragma unroll
        for (int k = 0; k < DEPTH; ++k) {
            const int64_t ek = e + (int64_t)k * NT * VEC;
            ok[k] = ek < p.d;
            e0[k] = (int)(ok[k] ? ek : 0);
            const int64_t at = base + e0[k];
            if constexpr (VECTOR) load_vec<T>(p.x, at, v[k]);
            else v[k][0] = load1<T>(p.x, at);
        }
        normalise_slots<T, A, DEPTH, VEC, VECTOR>(p, base, e0, ok, v, m.mean, m.m2);
    }
}

// --------------------------------------------------------------------------
// Host side.
template <class T, class A, int LPR, int NV, bool VECTOR>
void go_wave(const LNArgsDev& p, hipStream_t s) {
    constexpr int rows_per_block = (256 / kWave) * (kWave / LPR);
    hipLaunchKernelGGL((ln_wave<T, A, LPR, NV, VECTOR>), dim3((unsigned)((p.rows + rows_per_block - 1) / rows_per_block)),
                       dim3(256), 0, s, p);
}
template <class T, class A, int NT, int NV, bool VECTOR>
void go_block(const LNArgsDev& p, hipStream_t s) {
    hipLaunchKernelGGL((ln_block<T, A, NT, NV, VECTOR>), dim3((unsigned)p.rows), dim3(NT), 0, s, p);
}

template <class T, class A, bool VECTOR>
const char* launch(const LNArgsDev& p, hipStream_t s) {
    constexpr int VEC = VECTOR ? T::vec : 1;
    const int64_t slots = (p.d + VEC - 1) / VEC;
#define KF_LN_WAVE(LPR, NV)                           \
    if (slots <= (int64_t)(LPR) * (NV)) {              \
        go_wave<T, A, LPR, NV, VECTOR>(p, s);          \
        return VECTOR ? "ln_wave_vec_lpr" #LPR "_nv" #NV : "ln_wave_scalar_lpr" #LPR "_nv" #NV; \
    }
#define KF_LN_BLOCK(NT, NV)                           \
    if (slots <= (int64_t)(NT) * (NV)) {               \
        go_block<T, A, NT, NV, VECTOR>(p, s);          \
        return VECTOR ? "ln_block_vec_nt" #NT "_nv" #NV : "ln_block_scalar_nt" #NT "_nv" #NV; \
    }
    KF_LN_WAVE(1, 1)
    KF_LN_WAVE(2, 1)
    KF_LN_WAVE(4, 1)
    KF_LN_WAVE(8, 1)
    KF_LN_WAVE(16, 1)
    KF_LN_WAVE(16, 2)
    KF_LN_WAVE(16, 4)
    KF_LN_WAVE(32, 4)
    // Rows of 129-192 slots (the SD3.5 width): two rows per wave measured
    // 9.4 us against 10.2 us for one (bf16 [2,4096,1536], no affine); with
    // affine registers it would drop to 3 waves per SIMD, so only then.
    if constexpr (std::is_same_v<A, NoAffine>) {
        KF_LN_WAVE(32, 6)
    }
    KF_LN_WAVE(64, 3)
    KF_LN_WAVE(64, 4)
    KF_LN_BLOCK(128, 3)
    KF_LN_BLOCK(256, 2)
    KF_LN_BLOCK(512, 2)
    KF_LN_BLOCK(1024, 2)
    KF_LN_BLOCK(1024, 4)
    KF_LN_BLOCK(1024, 8)
#undef KF_LN_WAVE
#undef KF_LN_BLOCK
    hipLaunchKernelGGL((ln_stream<T, A, 1024, VECTOR>), dim3((unsigned)p.rows), dim3(1024), 0, s, p);
    return VECTOR ? "ln_stream_vec" : "ln_stream_scalar";
}

template <class T, class A>
kf_status run(const LayerNormArgs& a, hipStream_t s, const char** variant) {
    if (a.rows > (int64_t)INT32_MAX || a.d > (int64_t)INT32_MAX) {
        set_error("layer_norm: %lld rows of %lld elements exceed the grid limit", (long long)a.rows,
                  (long long)a.d);
        return KF_ERR_UNSUPPORTED_LAYOUT;
    }
    const LNArgsDev p{a.x, a.y, a.weight, a.bias, a.rows, (int32_t)a.d, a.eps};
    // 16-byte access needs whole vectors of x, y and the affine parameters
    // per row and 16-byte aligned bases.
    const int avec = (a.at == KF_FLOAT32) ? 4 : 8;
    const bool vec = (a.d % T::vec == 0) && (a.d % avec == 0) && ((uintptr_t)a.x % 16 == 0) &&
                     ((uintptr_t)a.y % 16 == 0) && ((uintptr_t)a.weight % 16 == 0) &&
                     ((uintptr_t)a.bias % 16 == 0);
    *variant = vec ? launch<T, A, true>(p, s) : launch<T, A, false>(p, s);
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) {
        set_error("layer_norm launch failed: %s", hipGetErrorString(err));
        return KF_ERR_HIP;
    }
    return KF_OK;
}

}  // namespace

kf_status layer_norm_launch(const LayerNormArgs& a, hipStream_t s, const char** variant) {
    const bool f32_affine = (a.at == KF_FLOAT32);
    const bool affine = a.weight || a.bias;
    switch (a.xt) {
        case KF_FLOAT32:
            return affine ? run<F32, F32>(a, s, variant) : run<F32, NoAffine>(a, s, variant);
        case KF_BFLOAT16:
            if (!affine) return run<BF16, NoAffine>(a, s, variant);
            return f32_affine ? run<BF16, F32>(a, s, variant) : run<BF16, BF16>(a, s, variant);
        case KF_FLOAT16:
            if (!affine) return run<F16, NoAffine>(a, s, variant);
            return f32_affine ? run<F16, F32>(a, s, variant) : run<F16, F16>(a, s, variant);
    }
    set_error("layer_norm: unsupported dtype");
    return KF_ERR_BAD_DTYPE;
}

}  // namespace kf
