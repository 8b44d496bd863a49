// kf_device.hpp -- gfx950 device primitives shared by the libkf355 kernels:
// 128-bit vector I/O with dtype conversion, and wave64 butterfly reductions
// built from DPP moves and the gfx950 permlane swaps (VALU only: no LDS
// traffic and no ds_bpermute).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kf {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// Element types.  `vec` is the number of elements in one 16-byte access.
struct F32 {
    static constexpr int bytes = 4;
    static constexpr int vec = 4;
};
struct BF16 {
    static constexpr int bytes = 2;
    static constexpr int vec = 8;
};
struct F16 {
    static constexpr int bytes = 2;
    static constexpr int vec = 8;
};

// Unpack one 32-bit word holding two 16-bit values (low half first).
__device__ __forceinline__ void unpack2(BF16, uint32_t w, float& a, float& b) {
    a = __uint_as_float(w << 16);
    b = __uint_as_float(w & 0xffff0000u);
}
__device__ __forceinline__ void unpack2(F16, uint32_t w, float& a, float& b) {
    f16x2 h = __builtin_bit_cast(f16x2, w);
    a = (float)h[0];
    b = (float)h[1];
}
// Pack two floats, each rounded to nearest-even (v_cvt_pk_bf16_f32 /
// v_cvt_pk_f16_f32 on gfx950).
__device__ __forceinline__ uint32_t pack2(BF16, float a, float b) {
    bf16x2 v = {(__bf16)a, (__bf16)b};
    return __builtin_bit_cast(uint32_t, v);
}
__device__ __forceinline__ uint32_t pack2(F16, float a, float b) {
    f16x2 v = {(_Float16)a, (_Float16)b};
    return __builtin_bit_cast(uint32_t, v);
}

// One 16-byte load.  With NT the load is non-temporal (the line is not kept
// for reuse), which is what an input read exactly once wants: measured on
// MI355X, a 256 MiB copy takes 84.9 us with non-temporal loads and stores
// against 87.4 us with non-temporal stores alone.
template <bool NT>
__device__ __forceinline__ u32x4 load16(const void* p) {
    if constexpr (NT) return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
    else return *reinterpret_cast<const u32x4*>(p);
}

// 16-byte vector load of T::vec elements at element offset `e` (e must be a
// multiple of T::vec and the address 16-byte aligned), widened to float.
template <class T, bool NT = false>
__device__ __forceinline__ void load_vec(const void* base, int64_t e, float* out) {
    const u32x4 v = load16<NT>(static_cast<const char*>(base) + e * T::bytes);
    if constexpr (T::vec == 4) {
#pragma unroll
        for (int i = 0; i < 4; ++i) out[i] = __uint_as_float(v[i]);
    } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) unpack2(T{}, v[i], out[2 * i], out[2 * i + 1]);
    }
}

// 16-byte vector store of T::vec elements, rounded to nearest-even.  With
// STREAM the store is non-temporal: the line is written to memory without
// being kept in cache, which is what an output that nothing re-reads wants
// (measured on MI355X: a 256 MiB copy takes ~30% less time with it).
__device__ __forceinline__ void put16(void* dst, u32x4 v, bool stream) {
    if (stream) __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(dst));
    else *reinterpret_cast<u32x4*>(dst) = v;
}
template <class T, bool STREAM = false>
__device__ __forceinline__ void store_vec(void* base, int64_t e, const float* in);
template <>
__device__ __forceinline__ void store_vec<F32, false>(void* base, int64_t e, const float* in) {
    u32x4 v;
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = __float_as_uint(in[i]);
    put16(static_cast<float*>(base) + e, v, false);
}
template <>
__device__ __forceinline__ void store_vec<F32, true>(void* base, int64_t e, const float* in) {
    u32x4 v;
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = __float_as_uint(in[i]);
    put16(static_cast<float*>(base) + e, v, true);
}
template <>
__device__ __forceinline__ void store_vec<BF16, false>(void* base, int64_t e, const float* in) {
    u32x4 v;
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = pack2(BF16{}, in[2 * i], in[2 * i + 1]);
    put16(static_cast<uint16_t*>(base) + e, v, false);
}
template <>
__device__ __forceinline__ void store_vec<BF16, true>(void* base, int64_t e, const float* in) {
    u32x4 v;
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = pack2(BF16{}, in[2 * i], in[2 * i + 1]);
    put16(static_cast<uint16_t*>(base) + e, v, true);
}
template <>
__device__ __forceinline__ void store_vec<F16, false>(void* base, int64_t e, const float* in) {
    u32x4 v;
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = pack2(F16{}, in[2 * i], in[2 * i + 1]);
    put16(static_cast<uint16_t*>(base) + e, v, false);
}
template <>
__device__ __forceinline__ void store_vec<F16, true>(void* base, int64_t e, const float* in) {
    u32x4 v;
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = pack2(F16{}, in[2 * i], in[2 * i + 1]);
    put16(static_cast<uint16_t*>(base) + e, v, true);
}

// Scalar element access (any alignment).
template <class T>
__device__ __forceinline__ float load1(const void* base, int64_t e);
template <>
__device__ __forceinline__ float load1<F32>(const void* base, int64_t e) {
    return static_cast<const float*>(base)[e];
}
template <>
__device__ __forceinline__ float load1<BF16>(const void* base, int64_t e) {
    return __uint_as_float(uint32_t(static_cast<const uint16_t*>(base)[e]) << 16);
}
template <>
__device__ __forceinline__ float load1<F16>(const void* base, int64_t e) {
    return (float)static_cast<const _Float16*>(base)[e];
}
template <class T>
__device__ __forceinline__ void store1(void* base, int64_t e, float v);
template <>
__device__ __forceinline__ void store1<F32>(void* base, int64_t e, float v) {
    static_cast<float*>(base)[e] = v;
}
template <>
__device__ __forceinline__ void store1<BF16>(void* base, int64_t e, float v) {
    static_cast<__bf16*>(base)[e] = (__bf16)v;
}
template <>
__device__ __forceinline__ void store1<F16>(void* base, int64_t e, float v) {
    static_cast<_Float16*>(base)[e] = (_Float16)v;
}

// ---------------------------------------------------------------------------
// Butterfly partner exchange.  Step s pairs each lane with one in the other
// half of its aligned block of 2^(s+1) lanes; after steps 0..k-1 every lane
// of an aligned block of 2^k lanes has combined the whole block.
//   s=0: quad_perm [1,0,3,2]      s=1: quad_perm [2,3,0,1]
//   s=2: row_half_mirror (i<->7-i within 8)
//   s=3: row_mirror      (i<->15-i within 16)
//   s=4: v_permlane16_swap (rows 0<->1, 2<->3)
//   s=5: v_permlane32_swap (halves 0<->1)
// Steps 2 and 3 pair a lane with a mirrored one rather than lane^4 / lane^8;
// that is still a butterfly because each quad (half-row) is already uniform.
template <int S>
__device__ __forceinline__ float partner(float v) {
    const int iv = __builtin_bit_cast(int, v);
    if constexpr (S == 0) {
        return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(iv, iv, 0xB1, 0xF, 0xF, false));
    } else if constexpr (S == 1) {
        return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(iv, iv, 0x4E, 0xF, 0xF, false));
    } else if constexpr (S == 2) {
        return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(iv, iv, 0x141, 0xF, 0xF, false));
    } else if constexpr (S == 3) {
        return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(iv, iv, 0x140, 0xF, 0xF, false));
    } else if constexpr (S == 4) {
        // After the swap, result[0] holds even rows duplicated, result[1] odd
        // rows duplicated: the partner is whichever differs from this lane's row.
        const unsigned u = __builtin_bit_cast(unsigned, v);
        auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
        const bool odd_row = (__lane_id() >> 4) & 1;
        return __builtin_bit_cast(float, odd_row ? r[0] : r[1]);
    } else {
        const unsigned u = __builtin_bit_cast(unsigned, v);
        auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
        const bool upper = __lane_id() >= 32;
        return __builtin_bit_cast(float, upper ? r[0] : r[1]);
    }
}

struct OpMax {
    __device__ __forceinline__ float operator()(float a, float b) const { return fmaxf(a, b); }
};
struct OpSum {
    __device__ __forceinline__ float operator()(float a, float b) const { return a + b; }
};

// Reduce over aligned groups of LANES lanes (a power of two <= 64); every
// lane of a group receives the group's result.  The combine must be
// commutative so that both lanes of a pair compute the same value.
template <int LANES, class Op>
__device__ __forceinline__ float group_reduce(float v, Op op) {
    if constexpr (LANES >= 2) v = op(v, partner<0>(v));
    if constexpr (LANES >= 4) v = op(v, partner<1>(v));
    if constexpr (LANES >= 8) v = op(v, partner<2>(v));
    if constexpr (LANES >= 16) v = op(v, partner<3>(v));
    if constexpr (LANES >= 32) v = op(v, partner<4>(v));
    if constexpr (LANES >= 64) v = op(v, partner<5>(v));
    return v;
}

// Uniform value of lane 0 (SGPR broadcast).
__device__ __forceinline__ float uniform0(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, v)));
}

// ---------------------------------------------------------------------------
// Moments (count, mean, M2) and their Chan et al. parallel combine, shared by
// GroupNorm and LayerNorm.
struct Moments {
    float n, mean, m2;
};

// Chan et al. combine of two partial moments (a before b).  The weight
// b.n / n uses the hardware reciprocal (v_rcp_f32, within 1 ulp; exact for
// power-of-two counts) instead of an IEEE division: the merges sit on the
// critical path between a workgroup's loads and its stores.
__device__ __forceinline__ Moments chan(Moments a, Moments b) {
    const float n = a.n + b.n;
    if (n == 0.f) return Moments{0.f, 0.f, 0.f};
    const float d = b.mean - a.mean;
    const float f = b.n * __builtin_amdgcn_rcpf(n);
    return Moments{n, fmaf(d, f, a.mean), a.m2 + b.m2 + d * d * a.n * f};
}

// Butterfly step S: the lane in the lower half of its aligned block of
// 2^(S+1) lanes is the left operand, so both lanes of a pair compute
// bit-identical results.
template <int S>
__device__ __forceinline__ Moments moments_step(Moments m) {
    Moments o{partner<S>(m.n), partner<S>(m.mean), partner<S>(m.m2)};
    const bool lower = (__lane_id() & (1 << S)) == 0;
    return lower ? chan(m, o) : chan(o, m);
}

// Combine over aligned groups of LANES lanes (a power of two <= 64); every
// lane of a group ends with the group's moments.
template <int LANES>
__device__ __forceinline__ Moments moments_group(Moments m) {
    if constexpr (LANES >= 2) m = moments_step<0>(m);
    if constexpr (LANES >= 4) m = moments_step<1>(m);
    if constexpr (LANES >= 8) m = moments_step<2>(m);
    if constexpr (LANES >= 16) m = moments_step<3>(m);
    if constexpr (LANES >= 32) m = moments_step<4>(m);
    if constexpr (LANES >= 64) m = moments_step<5>(m);
    return m;
}

__device__ __forceinline__ Moments moments_wave(Moments m) { return moments_group<kWave>(m); }

// Workgroup-wide combine of NW waves: butterfly inside each wave, then the
// waves in index order through LDS (`lds` holds NW entries).  Every thread
// gets the result.
template <int NW>
__device__ __forceinline__ Moments moments_block(Moments m, Moments* lds) {
    m = moments_wave(m);
    const int w = threadIdx.x / kWave;
    if ((threadIdx.x & (kWave - 1)) == 0) lds[w] = m;
    __syncthreads();
    Moments t = lds[0];
#pragma unroll
    for (int i = 1; i < NW; ++i) t = chan(t, lds[i]);
    __syncthreads();
    return t;
}

}  // namespace kf
