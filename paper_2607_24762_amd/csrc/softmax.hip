// softmax.hip -- row softmax for gfx950 (PyTorch `softmax(x, dim)` semantics,
// the operator behind the paper's Gemma 4 E2B and Qwen 3.5 softmax results,
// Section IV-C).
//
// Every variant makes one pass over HBM for reading and one for writing when
// the row fits on chip:
//   sm_wave   LPR lanes own a row (LPR = 1..64, so 64/LPR rows per wave); the
//             row stays in registers; max and sum are butterfly reductions
//             inside the lane group; no LDS, no barriers.
//   sm_block  one workgroup owns a row held in registers; per-wave partials
//             are combined through LDS.
//   sm_stream one workgroup per row of any length: an online (max, sum) pass,
//             then a write pass that reads the row again.
//   sm_span   short rows that are not whole 16-byte vectors (e.g. 257
//             router logits): R consecutive rows, chosen so that their span
//             starts 16-byte aligned for input and output, are staged in LDS
//             with 16-byte loads; LPR lanes per row reduce and normalise in
//             LDS; the span is written back with 16-byte stores.
//   sm_wave_edge / sm_block_edge  longer rows that are not whole vectors,
//             on aligned bases: the aligned 16-byte vectors covering the row,
//             neighbouring rows' elements masked, the two end vectors
//             written element by element.
//   sm_causal / sm_causal_edge / sm_causal_stream  the scaled causal
//             softmax of eager attention: the resident kernels' layouts,
//             and for longer rows the two-pass stream (whole or masked
//             16-byte vectors on aligned bases), each reading only the
//             visible prefix of a row.
//   sm_cols   softmax over a non-innermost axis: one thread per column,
//             online pass then write pass, coalesced across the inner axis.
#include <math.h>
#include <stdio.h>

#include <array>

#include <type_traits>
#include <utility>

#include "kf_device.hpp"
#include "kf_exchange.hpp"
#include "kf_internal.h"

namespace kf {
namespace {

constexpr float kLog2e = 1.4426950408889634f;

// e^(x - m) as 2^((x - m) * log2 e): subtracting first keeps x == m exact
// (2^0 = 1), so a uniform row gives exactly 1/L and a one-hot row exactly 1.
// Used for ratios of exponentials (the online merge).
__device__ __forceinline__ float exp_rel(float x, float m) {
    return __builtin_amdgcn_exp2f((x - m) * kLog2e);
}

// Per-element exponential for output type TO, scaled by 2^SHIFT: the factor
// cancels in y = e / sum(e).  The hardware exp2 (v_exp_f32) flushes results
// below 2^-126.  Only a bf16 output can represent such values (its smallest
// subnormal is 2^-133; fp16's is 2^-24 and fp32 outputs are judged by an
// absolute bound), and since sum(e) >= 2^SHIFT every y >= 2^-134 comes from
// an exponent >= -134: with SHIFT = 8 all of those are computed as normal
// numbers, and the final multiply by 1/sum produces the subnormal exactly.
// The shift costs nothing: it rides in the fma.
template <class TO>
struct Shift {
    static constexpr float value = 0.f;
};
template <>
struct Shift<BF16> {
    static constexpr float value = 8.f;
};
template <class TO>
__device__ __forceinline__ float exp_out(float x, float m) {
    if constexpr (Shift<TO>::value == 0.f) return __builtin_amdgcn_exp2f((x - m) * kLog2e);
    else return __builtin_amdgcn_exp2f(fmaf(x - m, kLog2e, Shift<TO>::value));
}

// Writes `n` floats (n * sizeof(TO) is a multiple of 16 bytes) starting at
// element e, as non-temporal 16-byte stores: softmax output is written once
// and not re-read by this kernel.
template <class TO, int N>
__device__ __forceinline__ void store_span(void* y, int64_t e, const float* v) {
    static_assert((N % TO::vec) == 0, "span must be whole vectors");
#pragma unroll
    for (int i = 0; i < N / TO::vec; ++i) store_vec<TO, true>(y, e + i * TO::vec, v + i * TO::vec);
}

// Sets slots outside the row (or of a row past the end) to -inf; slot k of
// lane-in-row `lr` starts at element (lr + k * STRIDE) * VEC.
template <int NV, int VEC, int STRIDE>
__device__ __forceinline__ void mask_slots(float (&v)[NV][VEC], int lr, bool row_ok, int32_t len) {
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        const bool ok = row_ok && (lr + k * STRIDE) * VEC < len;
#pragma unroll
        for (int i = 0; i < VEC; ++i) v[k][i] = ok ? v[k][i] : -INFINITY;
    }
}

// --------------------------------------------------------------------------
// Register-resident rows, LPR lanes per row.
template <class TI, class TO, int LPR, int NV, bool VECTOR>
__global__ __launch_bounds__(256) void sm_wave(const void* __restrict__ x, void* __restrict__ y,
                                               int64_t rows, int32_t len) {
    constexpr int VEC = VECTOR ? TI::vec : 1;
    constexpr int RPW = kWave / LPR;
    const int lane = threadIdx.x & (kWave - 1);
    const int lr = lane & (LPR - 1);
    const int64_t row = ((int64_t)blockIdx.x * (blockDim.x / kWave) + (threadIdx.x / kWave)) * RPW + lane / LPR;
    const bool row_ok = row < rows;
    const int64_t base = row * (int64_t)len;

    // Every slot is loaded unconditionally (an out-of-range slot re-reads
    // element 0, which always exists) so the loads issue back to back with no
    // wait between them; out-of-range slots are then set to -inf, in a branch
    // taken only by waves that have any.
    float v[NV][VEC];
    const bool full = row_ok && (LPR * NV * VEC == len);
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        const int e0 = (lr + k * LPR) * VEC;
        const int64_t at = (row_ok && e0 < len) ? base + e0 : 0;
        if constexpr (VECTOR) load_vec<TI, true>(x, at, v[k]);
        else v[k][0] = load1<TI>(x, at);
    }
    if (!__all(full)) mask_slots<NV, VEC, LPR>(v, lr, row_ok, len);
    float m = -INFINITY;
#pragma unroll
    for (int k = 0; k < NV; ++k)
#pragma unroll
        for (int i = 0; i < VEC; ++i) m = fmaxf(m, v[k][i]);
    m = group_reduce<LPR>(m, OpMax{});

    float s = 0.f;
#pragma unroll
    for (int k = 0; k < NV; ++k)
#pragma unroll
        for (int i = 0; i < VEC; ++i) {
            v[k][i] = exp_out<TO>(v[k][i], m);
            s += v[k][i];
        }
    s = group_reduce<LPR>(s, OpSum{});
    const float inv = 1.f / s;

#pragma unroll
    for (int k = 0; k < NV; ++k) {
        const int e0 = (lr + k * LPR) * VEC;
        if (row_ok && e0 < len) {
#pragma unroll
            for (int i = 0; i < VEC; ++i) v[k][i] *= inv;
            if constexpr (VECTOR) store_span<TO, VEC>(y, base + e0, v[k]);
            else store1<TO>(y, base + e0, v[k][0]);
        }
    }
}

// --------------------------------------------------------------------------
// Register-resident rows, one workgroup of NT threads per row.
template <int NW, class Op>
__device__ __forceinline__ float block_reduce(float v, Op op, float* red) {
    v = group_reduce<kWave>(v, op);
    const int w = threadIdx.x / kWave;
    if ((threadIdx.x & (kWave - 1)) == 0) red[w] = v;
    __syncthreads();
    float r = red[0];
#pragma unroll
    for (int i = 1; i < NW; ++i) r = op(r, red[i]);
    __syncthreads();  // red[] is reused by the next reduction
    return r;
}

template <class TI, class TO, int NT, int NV, bool VECTOR>
__global__ __launch_bounds__(NT) void sm_block(const void* __restrict__ x, void* __restrict__ y,
                                               int32_t len) {
    constexpr int VEC = VECTOR ? TI::vec : 1;
    constexpr int NW = NT / kWave;
    __shared__ float red[NW];
    const int64_t base = (int64_t)blockIdx.x * len;
    // Each wave owns a contiguous segment of NV*64 slots (slot k of lane l
    // of wave w is w*NV*64 + k*64 + l): every wave streams one contiguous
    // stretch of the row, the pattern that moves HBM fastest on this part.
    const int lane = threadIdx.x & (kWave - 1);
    const int seg = (threadIdx.x / kWave) * NV * kWave + lane;

    // Unconditional loads (out-of-range slots re-read the row's first
    // element), then masking, as in sm_wave.
    float v[NV][VEC];
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        const int e0 = (seg + k * kWave) * VEC;
        const int64_t at = base + (e0 < len ? e0 : 0);
        if constexpr (VECTOR) load_vec<TI, true>(x, at, v[k]);
        else v[k][0] = load1<TI>(x, at);
    }
    if (NT * NV * VEC != len) mask_slots<NV, VEC, kWave>(v, seg, true, len);
    float m = -INFINITY;
#pragma unroll
    for (int k = 0; k < NV; ++k)
#pragma unroll
        for (int i = 0; i < VEC; ++i) m = fmaxf(m, v[k][i]);
    m = block_reduce<NW>(m, OpMax{}, red);

    float s = 0.f;
#pragma unroll
    for (int k = 0; k < NV; ++k)
#pragma unroll
        for (int i = 0; i < VEC; ++i) {
            v[k][i] = exp_out<TO>(v[k][i], m);
            s += v[k][i];
        }
    s = block_reduce<NW>(s, OpSum{}, red);
    const float inv = 1.f / s;

#pragma unroll
    for (int k = 0; k < NV; ++k) {
        const int e0 = (seg + k * kWave) * VEC;
        if (e0 < len) {
#pragma unroll
            for (int i = 0; i < VEC; ++i) v[k][i] *= inv;
            if constexpr (VECTOR) store_span<TO, VEC>(y, base + e0, v[k]);
            else store1<TO>(y, base + e0, v[k][0]);
        }
    }
}

// --------------------------------------------------------------------------
// Rows that are not whole 16-byte vectors (len >= TI::vec, both bases
// 16-byte aligned).  A row [r0, r1) is covered by the aligned vectors from
// the one at or below r0: slot s of the row is the vector at
// a0 + s * VEC, a0 = floor(r0 / VEC) * VEC, so every load is a 16-byte load
// and at most ceil((len - 1) / VEC) + 1 slots are needed.  Elements of the
// neighbouring rows in the two end vectors are set to -inf after the loads
// (they weigh nothing), and only the row's own elements are written: whole
// vectors inside the row with 16-byte stores, the two end vectors element by
// element, so two rows sharing a vector never overwrite each other's values.

// Loads slots s0 + k * STRIDE (k < NV) of the row (elements [lo, hi)
// relative to a0), multiplied by `scale` when SCALED.  Offsets are 32-bit,
// relative to a0 (the row spans fewer than 2^31 elements): lo and hi are
// the row's bounds and room the elements left in the tensor from a0.  Every
// vector load is issued unconditionally: a slot past the row, a vector
// crossing the end of the tensor, or a row past the last reads the vector at
// a0 (for a row past the last, a0 = 0), which lies inside the tensor because
// len >= VEC.  The tensor's last vector, when partial, is then read element
// by element.
template <class TI, int NV, int STRIDE, bool SCALED = false>
__device__ __forceinline__ void edge_load(const void* x, int64_t a0, int s0, int32_t lo, int32_t hi,
                                          int32_t room, bool row_ok, float (&v)[NV][TI::vec],
                                          float scale = 1.f) {
    constexpr int VEC = TI::vec;
    const void* xa = static_cast<const char*>(x) + a0 * TI::bytes;
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        const int32_t e = (s0 + k * STRIDE) * VEC;
        const bool use = row_ok && e < hi && e <= room - VEC;
        load_vec<TI>(xa, use ? e : 0, v[k]);  // not non-temporal: neighbouring rows share the end vectors
    }
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        const int32_t e = (s0 + k * STRIDE) * VEC;
        if (row_ok && e < hi && e > room - VEC) {
#pragma unroll
            for (int i = 0; i < VEC; ++i)
                if (e + i < hi) v[k][i] = load1<TI>(xa, e + i);
        }
#pragma unroll
        for (int i = 0; i < VEC; ++i) {
            const float z = SCALED ? v[k][i] * scale : v[k][i];
            v[k][i] = (row_ok && e + i >= lo && e + i < hi) ? z : -INFINITY;
        }
    }
}

// Scales slots s0 + k * STRIDE by inv and writes the row's own elements.
template <class TO, int VEC, int NV, int STRIDE>
__device__ __forceinline__ void edge_store(void* y, int64_t a0, int s0, int32_t lo, int32_t hi, bool row_ok,
                                           float (&v)[NV][VEC], float inv) {
    void* ya = static_cast<char*>(y) + a0 * TO::bytes;
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        const int32_t e = (s0 + k * STRIDE) * VEC;
        if (row_ok && e < hi) {
#pragma unroll
            for (int i = 0; i < VEC; ++i) v[k][i] *= inv;
            if (e >= lo && e + VEC <= hi) {
                store_span<TO, VEC>(ya, e, v[k]);
            } else {
#pragma unroll
                for (int i = 0; i < VEC; ++i)
                    if (e + i >= lo && e + i < hi) store1<TO>(ya, e + i, v[k][i]);
            }
        }
    }
}

// Row bounds relative to its first aligned vector, and the elements left in
// the tensor from there (capped at 2^31 - 1).
struct EdgeRow {
    int64_t a0;
    int32_t lo, hi, room;
    template <int VEC>
    __device__ __forceinline__ static EdgeRow make(int64_t r0, int32_t len, int64_t total, bool row_ok) {
        EdgeRow r;
        r.a0 = row_ok ? (r0 / VEC) * VEC : 0;
        r.lo = (int32_t)(r0 - r.a0);
        r.hi = r.lo + len;
        const int64_t left = total - r.a0;
        r.room = left < (int64_t)INT32_MAX ? (int32_t)left : INT32_MAX;
        return r;
    }
};

// sm_wave for such rows: LPR lanes own a row, lane lr holds slots
// lr + k * LPR.
template <class TI, class TO, int LPR, int NV>
__global__ __launch_bounds__(256) void sm_wave_edge(const void* __restrict__ x, void* __restrict__ y,
                                                    int64_t rows, int32_t len) {
    constexpr int VEC = TI::vec;
    constexpr int RPW = kWave / LPR;
    const int lane = threadIdx.x & (kWave - 1);
    const int lr = lane & (LPR - 1);
    const int64_t row = ((int64_t)blockIdx.x * (blockDim.x / kWave) + (threadIdx.x / kWave)) * RPW + lane / LPR;
    const bool row_ok = row < rows;
    const EdgeRow er = EdgeRow::make<VEC>(row * (int64_t)len, len, rows * (int64_t)len, row_ok);

    float v[NV][VEC];
    edge_load<TI, NV, LPR>(x, er.a0, lr, er.lo, er.hi, er.room, row_ok, v);
    float m = -INFINITY;
#pragma unroll
    for (int k = 0; k < NV; ++k)
#pragma unroll
        for (int i = 0; i < VEC; ++i) m = fmaxf(m, v[k][i]);
    m = group_reduce<LPR>(m, OpMax{});
    float s = 0.f;
#pragma unroll
    for (int k = 0; k < NV; ++k)
#pragma unroll
        for (int i = 0; i < VEC; ++i) {
            v[k][i] = exp_out<TO>(v[k][i], m);
            s += v[k][i];
        }
    s = group_reduce<LPR>(s, OpSum{});
    edge_store<TO, VEC, NV, LPR>(y, er.a0, lr, er.lo, er.hi, row_ok, v, 1.f / s);
}

// sm_block for such rows: one workgroup per row, each wave owning NV * 64
// consecutive slots.
template <class TI, class TO, int NT, int NV>
__global__ __launch_bounds__(NT) void sm_block_edge(const void* __restrict__ x, void* __restrict__ y,
                                                    int32_t len) {
    constexpr int VEC = TI::vec;
    constexpr int NW = NT / kWave;
    __shared__ float red[NW];
    const EdgeRow er = EdgeRow::make<VEC>((int64_t)blockIdx.x * len, len, (int64_t)gridDim.x * len, true);
    const int seg = (threadIdx.x / kWave) * NV * kWave + (threadIdx.x & (kWave - 1));

    float v[NV][VEC];
    edge_load<TI, NV, kWave>(x, er.a0, seg, er.lo, er.hi, er.room, true, v);
    float m = -INFINITY;
#pragma unroll
    for (int k = 0; k < NV; ++k)
#pragma unroll
        for (int i = 0; i < VEC; ++i) m = fmaxf(m, v[k][i]);
    m = block_reduce<NW>(m, OpMax{}, red);
    float s = 0.f;
#pragma unroll
    for (int k = 0; k < NV; ++k)
#pragma unroll
        for (int i = 0; i < VEC; ++i) {
            v[k][i] = exp_out<TO>(v[k][i], m);
            s += v[k][i];
        }
    s = block_reduce<NW>(s, OpSum{}, red);
    edge_store<TO, VEC, NV, kWave>(y, er.a0, seg, er.lo, er.hi, true, v, 1.f / s);
}

// --------------------------------------------------------------------------
// Rows of `len` elements that are not whole 16-byte vectors, R rows per
// workgroup (R * len <= TILE floats, R a multiple of what makes r0 * len a
// whole number of input and output vectors, so every span starts aligned).
constexpr int kSpanFloats = 4096;      // staging that decides whether spans apply: 16 KiB of fp32

template <class TI, class TO, int LPR, int NPL, int TILE>
__global__ __launch_bounds__(256) void sm_span(const void* __restrict__ x, void* __restrict__ y, int64_t rows,
                                               int32_t len, int32_t R) {
    extern __shared__ float4 tile4[];  // R * len floats
    float* tile = reinterpret_cast<float*>(tile4);
    const int64_t r0 = (int64_t)blockIdx.x * R;
    const int32_t nr = (int32_t)((rows - r0) < R ? (rows - r0) : R);
    const int32_t span = nr * len;
    const int64_t base = r0 * len;

    // Stage: whole input vectors first (all loads before the LDS stores),
    // then the span's last partial vector element by element.
    constexpr int VI = TI::vec;
    constexpr int NL = (TILE + 256 * VI - 1) / (256 * VI);
    const int32_t whole_in = span - span % VI;
    float v[NL][VI];
#pragma unroll
    for (int k = 0; k < NL; ++k) {
        const int32_t e = (k * 256 + (int)threadIdx.x) * VI;
        if (e < whole_in) load_vec<TI, true>(x, base + e, v[k]);
    }
#pragma unroll
    for (int k = 0; k < NL; ++k) {
        const int32_t e = (k * 256 + (int)threadIdx.x) * VI;
        if (e < whole_in) {
#pragma unroll
            for (int i = 0; i < VI; i += 4)
                tile4[(e + i) / 4] = make_float4(v[k][i], v[k][i + 1], v[k][i + 2], v[k][i + 3]);
        }
    }
    for (int32_t e = whole_in + threadIdx.x; e < span; e += 256) tile[e] = load1<TI>(x, base + e);
    __syncthreads();

    // Row q: elements lr, lr + LPR, ... (at most NPL of them; the planner
    // picks NPL at most 3 above ceil(len / LPR), since every slot costs an
    // LDS read and an exponential) of the LPR lanes that own it, read from
    // LDS into registers in one batch (slots past the row are -inf), reduced
    // and normalised there, written back once.  Lanes of rows past nr take
    // part in the reductions and write nothing.
    const int q = threadIdx.x / LPR, lr = threadIdx.x % LPR;
    const bool row_ok = q < nr;
    float* row = tile + (row_ok ? q : 0) * len;
    float v2[NPL];
#pragma unroll
    for (int k = 0; k < NPL; ++k) {
        const int32_t e = lr + k * LPR;
        v2[k] = (row_ok && e < len) ? row[e] : -INFINITY;
    }
    float m = -INFINITY;
#pragma unroll
    for (int k = 0; k < NPL; ++k) m = fmaxf(m, v2[k]);
    m = group_reduce<LPR>(m, OpMax{});
    float sum = 0.f;
#pragma unroll
    for (int k = 0; k < NPL; ++k) {
        v2[k] = exp_out<TO>(v2[k], m);
        sum += v2[k];
    }
    sum = group_reduce<LPR>(sum, OpSum{});
    const float inv = 1.f / sum;
#pragma unroll
    for (int k = 0; k < NPL; ++k) {
        const int32_t e = lr + k * LPR;
        if (row_ok && e < len) row[e] = v2[k] * inv;
    }
    __syncthreads();

    // Store the span: whole output vectors, then the partial tail.
    constexpr int VO = TO::vec;
    const int32_t whole_out = span - span % VO;
    for (int32_t e = (int32_t)threadIdx.x * VO; e < whole_out; e += 256 * VO) {
        float o[VO];
#pragma unroll
        for (int i = 0; i < VO; ++i) o[i] = tile[e + i];
        store_vec<TO, true>(y, base + e, o);
    }
    for (int32_t e = whole_out + threadIdx.x; e < span; e += 256) store1<TO>(y, base + e, tile[e]);
}

// --------------------------------------------------------------------------
// Scaled causal softmax over rows of [batch * q, k]: query i = row % q sees
// keys j < live = clamp(i + k - q + 1, 0, k).  One workgroup per row with
// wave-contiguous segments as in sm_block; a wave whose whole segment is
// masked issues no loads, so the masked triangle is never read, and every
// slot is written (masked keys give exp(-inf) = +0).  A row with no visible
// key has max -inf and comes out NaN, as the masked softmax definition does.
template <class TI, class TO, int NT, int NV, bool VECTOR>
__global__ __launch_bounds__(NT) void sm_causal(const void* __restrict__ x, void* __restrict__ y, int32_t q,
                                                int32_t k, float scale) {
    constexpr int VEC = VECTOR ? TI::vec : 1;
    constexpr int NW = NT / kWave;
    __shared__ float red[NW];
    const int64_t row = blockIdx.x;
    const int32_t i = (int32_t)(row % q);
    const int32_t live = max(0, min(k, i + (k - q) + 1));
    const int64_t base = row * k;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int seg = wave * NV * kWave + lane;

    float v[NV][VEC];
    if (wave * NV * kWave * VEC < live) {  // uniform per wave
#pragma unroll
        for (int kk = 0; kk < NV; ++kk) {
            const int e0 = (seg + kk * kWave) * VEC;
            const int64_t at = base + (e0 < live ? e0 : 0);
            if constexpr (VECTOR) load_vec<TI, true>(x, at, v[kk]);
            else v[kk][0] = load1<TI>(x, at);
        }
#pragma unroll
        for (int kk = 0; kk < NV; ++kk) {
            const int e0 = (seg + kk * kWave) * VEC;
#pragma unroll
            for (int ii = 0; ii < VEC; ++ii) v[kk][ii] = (e0 + ii < live) ? v[kk][ii] * scale : -INFINITY;
        }
    } else {
#pragma unroll
        for (int kk = 0; kk < NV; ++kk)
#pragma unroll
            for (int ii = 0; ii < VEC; ++ii) v[kk][ii] = -INFINITY;
    }
    float m = -INFINITY;
#pragma unroll
    for (int kk = 0; kk < NV; ++kk)
#pragma unroll
        for (int ii = 0; ii < VEC; ++ii) m = fmaxf(m, v[kk][ii]);
    m = block_reduce<NW>(m, OpMax{}, red);

    float s = 0.f;
#pragma unroll
    for (int kk = 0; kk < NV; ++kk)
#pragma unroll
        for (int ii = 0; ii < VEC; ++ii) {
            v[kk][ii] = exp_out<TO>(v[kk][ii], m);
            s += v[kk][ii];
        }
    s = block_reduce<NW>(s, OpSum{}, red);
    const float inv = 1.f / s;

#pragma unroll
    for (int kk = 0; kk < NV; ++kk) {
        const int e0 = (seg + kk * kWave) * VEC;
        if (e0 < k) {
#pragma unroll
            for (int ii = 0; ii < VEC; ++ii) v[kk][ii] *= inv;
            if constexpr (VECTOR) store_span<TO, VEC>(y, base + e0, v[kk]);
            else store1<TO>(y, base + e0, v[kk][0]);
        }
    }
}

// sm_causal for rows that are not whole vectors (k >= TI::vec, aligned
// bases): the masked-vector row layout of sm_block_edge, with the visible
// prefix [lo, lo + live) loaded (scaled, masked to -inf past it) and every
// element of the row [lo, hi) written.
template <class TI, class TO, int NT, int NV>
__global__ __launch_bounds__(NT) void sm_causal_edge(const void* __restrict__ x, void* __restrict__ y, int32_t q,
                                                     int32_t k, float scale) {
    constexpr int VEC = TI::vec;
    constexpr int NW = NT / kWave;
    __shared__ float red[NW];
    const int64_t row = blockIdx.x;
    const int32_t i = (int32_t)(row % q);
    const int32_t live = max(0, min(k, i + (k - q) + 1));
    const EdgeRow er = EdgeRow::make<VEC>(row * k, k, (int64_t)gridDim.x * k, true);
    const int wave = threadIdx.x / kWave;
    const int seg = wave * NV * kWave + (threadIdx.x & (kWave - 1));
    const int32_t vis = er.lo + live;

    float v[NV][VEC];
    if (wave * NV * kWave * VEC < vis) {  // uniform per wave: segments past the visible prefix load nothing
        edge_load<TI, NV, kWave, true>(x, er.a0, seg, er.lo, vis, er.room, true, v, scale);
    } else {
#pragma unroll
        for (int kk = 0; kk < NV; ++kk)
#pragma unroll
            for (int ii = 0; ii < VEC; ++ii) v[kk][ii] = -INFINITY;
    }
    float m = -INFINITY;
#pragma unroll
    for (int kk = 0; kk < NV; ++kk)
#pragma unroll
        for (int ii = 0; ii < VEC; ++ii) m = fmaxf(m, v[kk][ii]);
    m = block_reduce<NW>(m, OpMax{}, red);
    float s = 0.f;
#pragma unroll
    for (int kk = 0; kk < NV; ++kk)
#pragma unroll
        for (int ii = 0; ii < VEC; ++ii) {
            v[kk][ii] = exp_out<TO>(v[kk][ii], m);
            s += v[kk][ii];
        }
    s = block_reduce<NW>(s, OpSum{}, red);
    edge_store<TO, VEC, NV, kWave>(y, er.a0, seg, er.lo, er.hi, true, v, 1.f / s);
}

// --------------------------------------------------------------------------
// Online normaliser state (m, s): s = sum of e^(x - m) over the elements
// seen.  A state with m = -inf has seen only -inf (or nothing) and weighs 0.
struct MS {
    float m, s;
};
__device__ __forceinline__ MS ms_merge(MS a, MS b) {
    const float mm = fmaxf(a.m, b.m);
    const float sa = (a.m == -INFINITY) ? 0.f : a.s * exp_rel(a.m, mm);
    const float sb = (b.m == -INFINITY) ? 0.f : b.s * exp_rel(b.m, mm);
    return MS{mm, sa + sb};
}
// Folds a chunk of n values into the state; s accumulates exp_out<TO>, so
// it carries the same 2^SHIFT factor as the write pass.
template <class TO, int N>
__device__ __forceinline__ MS ms_add(MS st, const float* v) {
    float cm = v[0];
#pragma unroll
    for (int i = 1; i < N; ++i) cm = fmaxf(cm, v[i]);
    const float mm = fmaxf(st.m, cm);
    if (mm == -INFINITY) return st;  // nothing but -inf so far
    float s = (st.m == -INFINITY) ? 0.f : st.s * exp_rel(st.m, mm);
#pragma unroll
    for (int i = 0; i < N; ++i) s += exp_out<TO>(v[i], mm);
    return MS{mm, s};
}
template <int S>
__device__ __forceinline__ MS ms_partner(MS a) {
    return MS{partner<S>(a.m), partner<S>(a.s)};
}
// Merge across a whole wave; ms_merge is commutative, so both lanes of a
// pair hold the same state after each step.
__device__ __forceinline__ MS ms_wave(MS a) {
    a = ms_merge(a, ms_partner<0>(a));
    a = ms_merge(a, ms_partner<1>(a));
    a = ms_merge(a, ms_partner<2>(a));
    a = ms_merge(a, ms_partner<3>(a));
    a = ms_merge(a, ms_partner<4>(a));
    a = ms_merge(a, ms_partner<5>(a));
    return a;
}

template <class TI, class TO, int NT, bool VECTOR>
__global__ __launch_bounds__(NT) void sm_stream(const void* __restrict__ x, void* __restrict__ y,
                                                int64_t len) {
    constexpr int VEC = VECTOR ? TI::vec : 1;
    constexpr int NW = NT / kWave;
    __shared__ float red_m[NW], red_s[NW];
    const int64_t base = (int64_t)blockIdx.x * len;

    // Pass 1: DEPTH loads in flight per thread per iteration; slots past the
    // end read as -inf, which ms_add ignores.
    constexpr int DEPTH = 4;
    MS st{-INFINITY, 0.f};
    for (int64_t e0 = (int64_t)threadIdx.x * VEC; e0 < len; e0 += (int64_t)DEPTH * NT * VEC) {
        float v[DEPTH * VEC];
#pragma unroll
        for (int d = 0; d < DEPTH; ++d) {
            const int64_t e = e0 + (int64_t)d * NT * VEC;
            if (e < len) {
                if constexpr (VECTOR) load_vec<TI>(x, base + e, v + d * VEC);
                else v[d] = load1<TI>(x, base + e);
            } else {
#pragma unroll
                for (int i = 0; i < VEC; ++i) v[d * VEC + i] = -INFINITY;
            }
        }
        st = ms_add<TO, DEPTH * VEC>(st, v);
    }
    st = ms_wave(st);
    const int w = threadIdx.x / kWave;
    if ((threadIdx.x & (kWave - 1)) == 0) {
        red_m[w] = st.m;
        red_s[w] = st.s;
    }
    __syncthreads();
    MS tot{red_m[0], red_s[0]};
#pragma unroll
    for (int i = 1; i < NW; ++i) tot = ms_merge(tot, MS{red_m[i], red_s[i]});
    // A row of only -inf keeps m = -inf, so x - m is NaN below: a NaN row,
    // as PyTorch gives.
    const float inv = 1.f / tot.s;

    for (int64_t e0 = (int64_t)threadIdx.x * VEC; e0 < len; e0 += (int64_t)DEPTH * NT * VEC) {
        float v[DEPTH][VEC];
#pragma unroll
        for (int d = 0; d < DEPTH; ++d) {
            const int64_t e = e0 + (int64_t)d * NT * VEC;
            if (e < len) {
                if constexpr (VECTOR) load_vec<TI>(x, base + e, v[d]);
                else v[d][0] = load1<TI>(x, base + e);
            }
        }
#pragma unroll
        for (int d = 0; d < DEPTH; ++d) {
            const int64_t e = e0 + (int64_t)d * NT * VEC;
            if (e < len) {
#pragma unroll
                for (int i = 0; i < VEC; ++i) v[d][i] = exp_out<TO>(v[d][i], tot.m) * inv;
                if constexpr (VECTOR) store_span<TO, VEC>(y, base + e, v[d]);
                else store1<TO>(y, base + e, v[d][0]);
            }
        }
    }
}

// --------------------------------------------------------------------------
// sm_causal for rows of any length: one workgroup per row, the online
// (max, sum) pass of sm_stream over the visible prefix only (the masked
// triangle is not read), then a write pass over the whole row that reads the
// prefix again.  Three access modes:
//   kStreamVec     rows of whole 16-byte vectors on aligned bases;
//   kStreamEdge    other rows on aligned bases, covered by the aligned
//                  vectors from the one at or below the row's start, as in
//                  sm_causal_edge: neighbouring rows' elements in the two end
//                  vectors are read and masked, only the row's own elements
//                  are written (whole vectors inside the row, the end vectors
//                  element by element), and a vector that would cross the end
//                  of the tensor is read element by element;
//   kStreamScalar  bases that are not 16-byte aligned: element by element.
// In-place safe: every element of the row is read and written by the same
// thread, the write pass after the barrier that ends the first; elements of
// a neighbouring row that an end vector reads are only ever masked.
constexpr int kStreamScalar = 0;
constexpr int kStreamVec = 1;
constexpr int kStreamEdge = 2;

template <class TI, class TO, int NT, int MODE>
__global__ __launch_bounds__(NT) void sm_causal_stream(const void* __restrict__ x, void* __restrict__ y, int64_t q,
                                                       int64_t k, float scale, int64_t total) {
    constexpr int VEC = MODE == kStreamScalar ? 1 : TI::vec;
    constexpr int NW = NT / kWave;
    constexpr int DEPTH = 4;
    constexpr int64_t STEP = (int64_t)DEPTH * NT * VEC;
    __shared__ float red_m[NW], red_s[NW];
    const int64_t row = blockIdx.x;
    const int64_t i = row % q;
    const int64_t live = i + (k - q) + 1 < 0 ? 0 : (i + (k - q) + 1 > k ? k : i + (k - q) + 1);
    // Loop offset e is tensor element a0 + e; the row's elements are
    // [lo, end) and its visible keys [lo, vis).
    const int64_t r0 = row * k;
    const int64_t a0 = MODE == kStreamEdge ? r0 / VEC * VEC : r0;
    const int64_t lo = r0 - a0, vis = lo + live, end = lo + k;
    const int64_t room = total - a0;  // tensor elements from a0 on
    auto load_slot = [&](int64_t e, float* v) {
        if constexpr (MODE == kStreamScalar) {
            v[0] = load1<TI>(x, a0 + e);
        } else if constexpr (MODE == kStreamVec) {
            load_vec<TI>(x, a0 + e, v);
        } else if (e + VEC <= room) {
            load_vec<TI>(x, a0 + e, v);
        } else {
#pragma unroll
            for (int ii = 0; ii < VEC; ++ii) v[ii] = e + ii < room ? load1<TI>(x, a0 + e + ii) : 0.f;
        }
    };

    // Elements [from, to) of the slot at e (clamped to [0, VEC]) lie in
    // [lo, bound): 32-bit compares per element.
    auto span = [&](int64_t e, int64_t bound, int& from, int& to) {
        const int64_t f = lo - e, t = bound - e;
        from = f < 0 ? 0 : (f > VEC ? VEC : (int)f);
        to = t < 0 ? 0 : (t > VEC ? VEC : (int)t);
    };

    MS st{-INFINITY, 0.f};
    for (int64_t e0 = (int64_t)threadIdx.x * VEC; e0 < vis; e0 += STEP) {
        float v[DEPTH * VEC];
#pragma unroll
        for (int d = 0; d < DEPTH; ++d) {
            const int64_t e = e0 + (int64_t)d * NT * VEC;
            if (e < vis) load_slot(e, v + d * VEC);
            int from, to;
            span(e, vis, from, to);
#pragma unroll
            for (int ii = 0; ii < VEC; ++ii)
                v[d * VEC + ii] = (ii >= from && ii < to) ? v[d * VEC + ii] * scale : -INFINITY;
        }
        st = ms_add<TO, DEPTH * VEC>(st, v);
    }
    st = ms_wave(st);
    const int w = threadIdx.x / kWave;
    if ((threadIdx.x & (kWave - 1)) == 0) {
        red_m[w] = st.m;
        red_s[w] = st.s;
    }
    __syncthreads();
    MS tot{red_m[0], red_s[0]};
#pragma unroll
    for (int j = 1; j < NW; ++j) tot = ms_merge(tot, MS{red_m[j], red_s[j]});
    // No visible key: m = -inf and every output is exp(-inf - -inf) = NaN.
    const float inv = 1.f / tot.s;

    for (int64_t e0 = (int64_t)threadIdx.x * VEC; e0 < end; e0 += STEP) {
        float v[DEPTH][VEC];
#pragma unroll
        for (int d = 0; d < DEPTH; ++d) {
            const int64_t e = e0 + (int64_t)d * NT * VEC;
            if (e < vis) load_slot(e, v[d]);
        }
#pragma unroll
        for (int d = 0; d < DEPTH; ++d) {
            const int64_t e = e0 + (int64_t)d * NT * VEC;
            if (e < end) {
                int from, to;
                span(e, vis, from, to);
#pragma unroll
                for (int ii = 0; ii < VEC; ++ii)
                    v[d][ii] = exp_out<TO>((ii >= from && ii < to) ? v[d][ii] * scale : -INFINITY, tot.m) * inv;
                if constexpr (MODE == kStreamScalar) {
                    store1<TO>(y, a0 + e, v[d][0]);
                } else if (MODE == kStreamVec || (e >= lo && e + VEC <= end)) {
                    store_span<TO, VEC>(y, a0 + e, v[d]);
                } else {
                    span(e, end, from, to);
#pragma unroll
                    for (int ii = 0; ii < VEC; ++ii)
                        if (ii >= from && ii < to) store1<TO>(y, a0 + e + ii, v[d][ii]);
                }
            }
        }
    }
}

// --------------------------------------------------------------------------
// Softmax over a non-innermost axis of [outer, len, inner]: thread per
// (outer, inner) column; neighbouring threads read neighbouring addresses.
template <class TI, class TO>
__global__ __launch_bounds__(256) void sm_cols(const void* __restrict__ x, void* __restrict__ y,
                                               int64_t outer, int64_t len, int64_t inner) {
    const int64_t col = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (col >= outer * inner) return;
    const int64_t o = col / inner, i = col - o * inner;
    const int64_t base = o * len * inner + i;
    constexpr int DEPTH = 4;
    MS st{-INFINITY, 0.f};
    for (int64_t j0 = 0; j0 < len; j0 += DEPTH) {
        float v[DEPTH];
#pragma unroll
        for (int d = 0; d < DEPTH; ++d) v[d] = (j0 + d < len) ? load1<TI>(x, base + (j0 + d) * inner) : -INFINITY;
        st = ms_add<TO, DEPTH>(st, v);
    }
    const float inv = 1.f / st.s;
    for (int64_t j = 0; j < len; ++j)
        store1<TO>(y, base + j * inner, exp_out<TO>(load1<TI>(x, base + j * inner), st.m) * inv);
}

// --------------------------------------------------------------------------
// Rows split over several workgroups (few long rows, such as decode-step
// attention scores [batch, heads, 1, kv]: one workgroup per row would leave
// most of the chip idle).  Part p of a row covers CH = 256 * NV * VEC flat
// elements starting at the 16-byte boundary at or below the row's start plus
// p * CH, so every load is an aligned 16-byte vector whatever the row length;
// elements outside the row are masked to -inf.  Each workgroup keeps its part
// in registers, reduces it to an online-normaliser state (m, s), exchanges
// that state with the other parts of its row (one 64-bit word each, see
// kf_exchange.hpp), merges all parts in part order and writes e^(x - M) / S
// straight from registers: one HBM read and one write, like sm_block.
constexpr int kSplitNT = 256;

struct SplitParams {
    const void* x;
    void* y;
    Exchange ex;    // one unit per row, ex.parts workgroups each
    int64_t len;    // row length
    int64_t total;  // elements in the tensor (rows * len)
};

// (m, s) as one never-zero word: m bits low, s bits high with the sign bit
// forced on (s is a sum of exponentials: never negative).
__device__ __forceinline__ uint64_t ms_encode(MS a) {
    return (uint64_t)__float_as_uint(a.m) | ((uint64_t)(__float_as_uint(a.s) | 0x80000000u) << 32);
}
__device__ __forceinline__ MS ms_decode(uint64_t w) {
    return MS{__uint_as_float((uint32_t)w), __uint_as_float((uint32_t)(w >> 32) & 0x7fffffffu)};
}

template <class TI, int NV>
struct SplitPart {
    static constexpr int VEC = TI::vec;
    static constexpr int NW = kSplitNT / kWave;
    static constexpr int64_t CH = (int64_t)kSplitNT * NV * VEC;
    float v[NV][VEC];

    // Flat index of the first element of slot k of this thread in part
    // `part` of the row starting at r0.  Each wave owns NV*64 consecutive
    // vectors of the part (the contiguous per-wave stream of sm_block).
    __device__ __forceinline__ static int64_t at(int64_t r0, int part, int k) {
        const int seg = (threadIdx.x / kWave) * NV * kWave + (threadIdx.x & (kWave - 1));
        return (r0 / VEC) * VEC + (int64_t)part * CH + (int64_t)(seg + k * kWave) * VEC;
    }

    // Loads the part and masks elements outside [r0, r0 + len) to -inf.  All
    // vector loads are issued unconditionally, from a clamped address when a
    // vector misses the row or crosses the tensor's end (the row's first
    // aligned vector, inside the tensor since len >= VEC); the rare edge
    // vectors are fixed up after every load is in flight.
    __device__ __forceinline__ void load(const SplitParams& p, int64_t r0, int part) {
        const int64_t r1 = r0 + p.len;
        const int64_t safe = (r0 / VEC) * VEC;
        bool edge = false;
#pragma unroll
        for (int k = 0; k < NV; ++k) {
            const int64_t e = at(r0, part, k);
            const bool use = e < r1 && e + VEC > r0 && e + VEC <= p.total;
            load_vec<TI, true>(p.x, use ? e : safe, v[k]);
            edge = edge || e < r0 || e + VEC > r1;
        }
        if (__any(edge)) {
#pragma unroll
            for (int k = 0; k < NV; ++k) {
                const int64_t e = at(r0, part, k);
                if (e < r1 && e + VEC > p.total) {  // the tensor's last, partial vector
#pragma unroll
                    for (int i = 0; i < VEC; ++i)
                        if (e + i < r1) v[k][i] = load1<TI>(p.x, e + i);
                }
#pragma unroll
                for (int i = 0; i < VEC; ++i) v[k][i] = (e + i >= r0 && e + i < r1) ? v[k][i] : -INFINITY;
            }
        }
    }

    // The part's (m, s); s accumulates exp_out<TO>, so it carries the same
    // 2^SHIFT factor as the write.  A part of only -inf (or none of the row)
    // gives (-inf, 0), which weighs nothing in the merge.  Block-uniform.
    template <class TO>
    __device__ __forceinline__ MS stats(float* red) const {
        float m = -INFINITY;
#pragma unroll
        for (int k = 0; k < NV; ++k)
#pragma unroll
            for (int i = 0; i < VEC; ++i) m = fmaxf(m, v[k][i]);
        m = block_reduce<NW>(m, OpMax{}, red);
        float s = 0.f;
        if (m != -INFINITY) {
#pragma unroll
            for (int k = 0; k < NV; ++k)
#pragma unroll
                for (int i = 0; i < VEC; ++i) s += exp_out<TO>(v[k][i], m);
        }
        s = block_reduce<NW>(s, OpSum{}, red);
        return MS{m, s};
    }

    template <class TO>
    __device__ __forceinline__ void store(const SplitParams& p, int64_t r0, int part, float mm, float inv) const {
        const int64_t r1 = r0 + p.len;
#pragma unroll
        for (int k = 0; k < NV; ++k) {
            const int64_t e = at(r0, part, k);
            float out[VEC];
#pragma unroll
            for (int i = 0; i < VEC; ++i) out[i] = exp_out<TO>(v[k][i], mm) * inv;
            if (e >= r0 && e + VEC <= r1) {
                store_span<TO, VEC>(p.y, e, out);
            } else {
#pragma unroll
                for (int i = 0; i < VEC; ++i)
                    if (e + i >= r0 && e + i < r1) store1<TO>(p.y, e + i, out[i]);
            }
        }
    }
};

template <class TI, class TO, int NV>
__global__ __launch_bounds__(kSplitNT) void sm_split(SplitParams p) {
    using P = SplitPart<TI, NV>;
    __shared__ float red[P::NW];
    __shared__ float stat[2];
    __shared__ int gathered;
    const int64_t row = blockIdx.x / p.ex.parts;
    const int part = (int)(blockIdx.x - row * p.ex.parts);
    const int64_t r0 = row * p.len;
    const int lane = threadIdx.x & (kWave - 1);

    P c;
    c.load(p, r0, part);
    const MS own = c.template stats<TO>(red);
    if (threadIdx.x < kWave) {
        if (threadIdx.x == 0) ex_publish(p.ex, row, part, ms_encode(own));
        // Lane l merges parts l, l+64, ... in order, then the wave merges
        // across lanes (ms_merge is exactly commutative, so every lane and
        // every workgroup of the row ends with the same bits).
        const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
        MS acc{-INFINITY, 0.f};
        bool all = true;
        for (int q = lane; q < p.ex.parts; q += kWave) {
            const uint64_t w = ex_poll(p.ex, row, q, t0, true);
            all = all && (w != 0);
            acc = ms_merge(acc, ms_decode(w));
        }
        acc = ms_wave(acc);
        const bool ok = __all(all);
        if (threadIdx.x == 0) {
            gathered = ok;
            stat[0] = acc.m;
            stat[1] = 1.f / acc.s;
        }
    }
    __syncthreads();
    if (!gathered) {
        // Some part of the row was not published in time (its workgroup is
        // not resident yet).  Recompute every part's state here with the
        // loads, thread mapping and arithmetic its owner uses and merge in
        // the same order: the result is bit-identical, so the kernel never
        // depends on co-residency.  (In-place calls are not split.)
        MS acc{-INFINITY, 0.f};
        for (int q = 0; q < p.ex.parts; ++q) {
            c.load(p, r0, q);
            const MS mq = c.template stats<TO>(red);
            if ((q & (kWave - 1)) == lane) acc = ms_merge(acc, mq);
        }
        if (threadIdx.x < kWave) {
            acc = ms_wave(acc);
            if (threadIdx.x == 0) {
                stat[0] = acc.m;
                stat[1] = 1.f / acc.s;
                ex_count_give_up(p.ex);
            }
        }
        c.load(p, r0, part);
        __syncthreads();
    }
    // Done reading the row's slots: count this workgroup out before the
    // stores, so the atomic's round trip overlaps them.  A row of only -inf
    // has M = -inf, so x - M is NaN: a NaN row, as the definition gives.
    unsigned before = 0;
    if (threadIdx.x == 0) before = ex_depart(p.ex, row);
    c.template store<TO>(p, r0, part, stat[0], stat[1]);
    if (threadIdx.x == 0) ex_leave(p.ex, row, before);
}

// --------------------------------------------------------------------------
// Variant selection.
template <class TI, class TO, int LPR, int NV, bool VECTOR>
void go_wave(const SoftmaxArgs& a, hipStream_t s) {
    constexpr int rows_per_block = (256 / kWave) * (kWave / LPR);
    const int64_t blocks = (a.outer + rows_per_block - 1) / rows_per_block;
    hipLaunchKernelGGL((sm_wave<TI, TO, LPR, NV, VECTOR>), dim3((unsigned)blocks), dim3(256), 0, s,
                       a.x, a.y, a.outer, (int32_t)a.len);
}
template <class TI, class TO, int NT, int NV, bool VECTOR>
void go_block(const SoftmaxArgs& a, hipStream_t s) {
    hipLaunchKernelGGL((sm_block<TI, TO, NT, NV, VECTOR>), dim3((unsigned)a.outer), dim3(NT), 0, s,
                       a.x, a.y, (int32_t)a.len);
}

struct Choice {
    void (*fn)(const SoftmaxArgs&, hipStream_t);
    const char* name;
};

// Smallest register-resident configuration whose capacity covers the row.
// Capacity = LPR * NV * VEC (lane groups) or NT * NV * VEC (workgroup per
// row) elements.  Vectorised rows wider than 256 slots (4 KiB of fp32 or
// bf16 pairs) go to a workgroup per row with two 16-byte slots per lane, so
// each wave streams 2 KiB of the row: measured on MI355X, a causal bf16
// [32768 x 4096] softmax takes 89.4 us that way against 92.0 us with one
// wave per row.  Unaligned (element-wise) rows stay on lane groups up to
// 1024 elements.
template <class TI, class TO, bool VECTOR>
Choice pick_resident(int64_t len) {
    constexpr int VEC = VECTOR ? TI::vec : 1;
    const int64_t slots = (len + VEC - 1) / VEC;
#define KF_WAVE(LPR, NV)                                                                       \
    if (slots <= (int64_t)(LPR) * (NV))                                                        \
        return Choice{go_wave<TI, TO, LPR, NV, VECTOR>, VECTOR ? "sm_wave_vec_lpr" #LPR "_nv" #NV \
                                                               : "sm_wave_scalar_lpr" #LPR "_nv" #NV};
#define KF_BLOCK(NT, NV)                                                                         \
    if (slots <= (int64_t)(NT) * (NV))                                                           \
        return Choice{go_block<TI, TO, NT, NV, VECTOR>, VECTOR ? "sm_block_vec_nt" #NT "_nv" #NV \
                                                               : "sm_block_scalar_nt" #NT "_nv" #NV};
    KF_WAVE(1, 1)
    KF_WAVE(2, 1)
    KF_WAVE(4, 1)
    KF_WAVE(8, 1)
    KF_WAVE(16, 1)
    KF_WAVE(16, 2)
    KF_WAVE(16, 4)
    KF_WAVE(32, 4)
    KF_WAVE(64, 4)
    if constexpr (VECTOR) {
        KF_BLOCK(256, 2)
        KF_BLOCK(512, 2)
        KF_BLOCK(1024, 2)
        KF_BLOCK(1024, 4)
        KF_BLOCK(1024, 8)
        if constexpr (TI::vec == 4) {
            KF_BLOCK(1024, 16)
        }
    } else {
        KF_WAVE(64, 8)
        KF_WAVE(64, 16)
        KF_BLOCK(256, 8)
        KF_BLOCK(512, 8)
        KF_BLOCK(1024, 8)
        KF_BLOCK(1024, 16)
    }
#undef KF_WAVE
#undef KF_BLOCK
    return Choice{nullptr, nullptr};
}

template <class TI, class TO, int LPR, int NV>
void go_wave_edge(const SoftmaxArgs& a, hipStream_t s) {
    constexpr int rows_per_block = (256 / kWave) * (kWave / LPR);
    const int64_t blocks = (a.outer + rows_per_block - 1) / rows_per_block;
    hipLaunchKernelGGL((sm_wave_edge<TI, TO, LPR, NV>), dim3((unsigned)blocks), dim3(256), 0, s, a.x, a.y, a.outer,
                       (int32_t)a.len);
}
template <class TI, class TO, int NT, int NV>
void go_block_edge(const SoftmaxArgs& a, hipStream_t s) {
    hipLaunchKernelGGL((sm_block_edge<TI, TO, NT, NV>), dim3((unsigned)a.outer), dim3(NT), 0, s, a.x, a.y,
                       (int32_t)a.len);
}

// Register-resident configuration for rows that are not whole vectors
// (bases 16-byte aligned, len >= TI::vec): the smallest whose slots cover
// the ceil((len - 1) / VEC) + 1 aligned vectors a row can touch.  Lane
// groups up to 256 slots, then a workgroup per row, as for whole-vector rows.
// The shortest rows that get here are 16-bit rows of more than 512 elements
// (shorter ones are staged spans), so lane groups start at 80 slots.
template <class TI, class TO>
Choice pick_edge(int64_t len) {
    constexpr int VEC = TI::vec;
    const int64_t slots = (len - 1 + VEC - 1) / VEC + 1;
#define KF_WAVE(LPR, NV)         \
    if (slots <= (int64_t)(LPR) * (NV)) \
        return Choice{go_wave_edge<TI, TO, LPR, NV>, "sm_wave_edge_lpr" #LPR "_nv" #NV};
#define KF_BLOCK(NT, NV)         \
    if (slots <= (int64_t)(NT) * (NV)) \
        return Choice{go_block_edge<TI, TO, NT, NV>, "sm_block_edge_nt" #NT "_nv" #NV};
    KF_WAVE(16, 5)
    KF_WAVE(32, 3)
    KF_WAVE(32, 4)
    KF_WAVE(32, 5)
    KF_WAVE(64, 3)
    KF_WAVE(64, 4)
    KF_BLOCK(256, 2)
    KF_BLOCK(256, 3)
    KF_BLOCK(512, 2)
    KF_BLOCK(512, 3)
    KF_BLOCK(1024, 2)
    KF_BLOCK(1024, 3)
    KF_BLOCK(1024, 4)
    KF_BLOCK(1024, 5)
    if constexpr (VEC == 4) {  // 16-element slots would spill at 9 per lane
        KF_BLOCK(1024, 9)
    }
#undef KF_WAVE
#undef KF_BLOCK
    return Choice{nullptr, nullptr};
}

// Launches sm_span with 16 lanes per row and exactly `slots` (9..32) slots
// per lane.  More than 16 slots only arise from rows of more than 256
// elements, whose 16 rows need a wider tile: at most 16 * 16 * slots floats,
// rounded up to whole 1024-float load rounds (so no load slot is issued that
// no element can fill: 5120 floats for 17 slots, where the full 8192 cost
// 1.2% on [16384, 257] fp32).
constexpr int span16_tile(int slots) { return slots <= 16 ? kSpanFloats : (slots + 3) / 4 * 1024; }
template <class TI, class TO, class Go, int... I>
void span_lanes16(int slots, Go& go, std::integer_sequence<int, I...>) {
    ((slots == I + 9 ? (go(sm_span<TI, TO, 16, I + 9, span16_tile(I + 9)>), 0) : 0), ...);
}

// sm_span for rows of `len` elements that are not whole vectors, when both
// bases are 16-byte aligned and at least the aligning row count fits
// kSpanFloats.  Returns false (nothing launched) otherwise.
//
// Rows of 129-512 elements: 16 rows per workgroup, 16 lanes per row (four
// rows per wave, the shape of the vector-row kernel on [16384, 256]), in up
// to 32 KiB of LDS.  Measured on [16384, L] fp32 against the plan below:
// L = 257 7.03 -> 6.33 us, 258 6.96 -> 6.30, 385 10.34 -> 8.52,
// 511 13.92 -> 10.57, 129 4.67 -> 4.22, 150 4.87 -> 4.47.  Other lengths:
// as many rows as fit 4096 floats, fewer while a lane would hold more than
// 16 of a row's elements (on [16384, 257] fp32: 12 rows and 17 per lane
// 8.27 us, 8 rows and 9 per lane 7.23 us, 4 rows and 5 per lane 8.88 us).
template <class TI, class TO>
bool run_span(const SoftmaxArgs& a, hipStream_t s, const char** variant) {
    if ((uintptr_t)a.x % 16 || (uintptr_t)a.y % 16 || a.len < 1 || a.len > kSpanFloats) return false;
    auto rows_for = [&](int64_t vec) {  // fewest rows whose span is a whole number of vectors
        int64_t r = 1;
        while ((a.len * r) % vec != 0) ++r;  // ends by r = vec
        return r;
    };
    const int64_t ra = rows_for(TI::vec), rb = rows_for(TO::vec);
    const int64_t align = ra > rb ? ra : rb;  // both are powers of two, so the larger is their lcm
    if (align * a.len > kSpanFloats) return false;
    auto lanes_for = [](int64_t rows) {  // the largest power of two <= 256 / rows, at most 64
        int l = 1;
        while (l < 64 && 2 * l * rows <= 256) l *= 2;
        return l;
    };
    int64_t R;
    if (a.len > 128 && a.len <= 512) {
        R = 16;  // align is at most 8, so 16 rows always start aligned
    } else {
        R = kSpanFloats / a.len;
        R = R > 256 ? 256 : R;
        R -= R % align;
        while (R - align >= align && (a.len + lanes_for(R) - 1) / lanes_for(R) > 16) R -= align;
    }
    const int lpr = lanes_for(R);
    const int64_t npl = (a.len + lpr - 1) / lpr;
    if (npl > 32) return false;
    const int64_t blocks = (a.outer + R - 1) / R;
    if (blocks > INT32_MAX) return false;
    const size_t lds = (size_t)(R * a.len) * sizeof(float);
    auto go = [&](auto kernel) {
        hipLaunchKernelGGL(kernel, dim3((unsigned)blocks), dim3(256), lds, s, a.x, a.y, a.outer, (int32_t)a.len,
                           (int32_t)R);
    };
    // Slots per lane: 8, 16 or 32, and on the 16-lane rows exactly
    // ceil(len / 16) from 9 up (on [16384, 257] fp32, 17 elements per lane:
    // 17 slots 6.35 us, 20 slots 6.49).
    int nplt = npl <= 8 ? 8 : npl <= 16 ? 16 : 32;
    if (lpr == 16 && npl > 8) nplt = (int)npl;
    auto with_npl = [&](auto lpr_tag) {
        constexpr int L = decltype(lpr_tag)::value;
        if (nplt == 8) go(sm_span<TI, TO, L, 8, kSpanFloats>);
        else if (nplt == 16) go(sm_span<TI, TO, L, 16, kSpanFloats>);
        else go(sm_span<TI, TO, L, 32, kSpanFloats>);
    };
    switch (lpr) {
        case 64: with_npl(std::integral_constant<int, 64>{}); break;
        case 32: with_npl(std::integral_constant<int, 32>{}); break;
        case 16:
            if (nplt == 8) go(sm_span<TI, TO, 16, 8, kSpanFloats>);
            else span_lanes16<TI, TO>(nplt, go, std::make_integer_sequence<int, 24>{});
            break;
        case 8: with_npl(std::integral_constant<int, 8>{}); break;
        case 4: with_npl(std::integral_constant<int, 4>{}); break;
        case 2: with_npl(std::integral_constant<int, 2>{}); break;
        default: with_npl(std::integral_constant<int, 1>{}); break;
    }
    // "sm_span_lpr<L>_npl<slots>" for L = 1..64 and slots = 1..32.
    static const auto names = [] {
        std::array<std::array<std::array<char, 24>, 33>, 7> t{};
        for (int li = 0; li < 7; ++li)
            for (int n = 1; n <= 32; ++n) snprintf(t[li][n].data(), t[li][n].size(), "sm_span_lpr%d_npl%d", 1 << li, n);
        return t;
    }();
    int li = 0;
    while ((1 << li) < lpr) ++li;
    *variant = names[li][nplt].data();
    return true;
}

template <class TI, class TO>
kf_status run(const SoftmaxArgs& a, hipStream_t s, const char** variant) {
    if (a.inner != 1) {
        const int64_t cols = a.outer * a.inner;
        const int64_t blocks = (cols + 255) / 256;
        if (blocks > INT32_MAX) {
            set_error("softmax: %lld columns exceed the grid limit", (long long)cols);
            return KF_ERR_UNSUPPORTED_LAYOUT;
        }
        hipLaunchKernelGGL((sm_cols<TI, TO>), dim3((unsigned)blocks), dim3(256), 0, s, a.x, a.y, a.outer,
                           a.len, a.inner);
        *variant = "sm_cols";
    } else {
        // Every kernel below puts at most one row per thread block index
        // group; keep the grid inside the 32-bit limit.
        if (a.outer > (int64_t)INT32_MAX) {
            set_error("softmax: %lld rows exceed the grid limit", (long long)a.outer);
            return KF_ERR_UNSUPPORTED_LAYOUT;
        }
        // 16-byte vectors need the row length to be whole vectors of both the
        // input and the output, and both base pointers 16-byte aligned.
        const bool vec_ok = (a.len % TI::vec == 0) && (a.len % TO::vec == 0) &&
                            ((uintptr_t)a.x % 16 == 0) && ((uintptr_t)a.y % 16 == 0);
        // Rows that are not whole vectors: staged spans where they apply;
        // otherwise, on 16-byte aligned bases, aligned vectors with masked
        // ends for 16-bit inputs (element-wise 2-byte loads move half the
        // bytes per instruction: bf16 [32768, 4097] 185 us element-wise,
        // 107 us with masked vectors) and for fp32 rows too long for the
        // element-wise resident kernels; fp32 rows within their reach stay
        // element-wise, which measured faster ([16384, 1025]: 26.6 against
        // 30.3 us).
        const bool edge_ok = !vec_ok && a.len >= TI::vec && ((uintptr_t)a.x % 16 == 0) &&
                             ((uintptr_t)a.y % 16 == 0) && a.len <= INT32_MAX;
        Choice c{nullptr, nullptr};
        if (!vec_ok && run_span<TI, TO>(a, s, variant)) {
            // staged spans launched
        } else {
            if (a.len <= INT32_MAX) {
                if (vec_ok) c = pick_resident<TI, TO, true>(a.len);
                else if (edge_ok && TI::vec == 8) c = pick_edge<TI, TO>(a.len);
                if (!c.fn && !vec_ok) c = pick_resident<TI, TO, false>(a.len);
                if (!c.fn && edge_ok) c = pick_edge<TI, TO>(a.len);
            }
            if (c.fn) {
                c.fn(a, s);
                *variant = c.name;
            } else if (vec_ok) {
                hipLaunchKernelGGL((sm_stream<TI, TO, 1024, true>), dim3((unsigned)a.outer), dim3(1024), 0, s,
                                   a.x, a.y, a.len);
                *variant = "sm_stream_vec";
            } else {
                hipLaunchKernelGGL((sm_stream<TI, TO, 1024, false>), dim3((unsigned)a.outer), dim3(1024), 0, s,
                                   a.x, a.y, a.len);
                *variant = "sm_stream_scalar";
            }
        }
    }
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) {
        set_error("softmax launch failed: %s", hipGetErrorString(err));
        return KF_ERR_HIP;
    }
    return KF_OK;
}

template <class TI, class TO, int NT, int NV, bool VECTOR>
void go_causal(const CausalSoftmaxArgs& a, hipStream_t s) {
    hipLaunchKernelGGL((sm_causal<TI, TO, NT, NV, VECTOR>), dim3((unsigned)(a.batch * a.q)), dim3(NT), 0, s, a.x,
                       a.y, (int32_t)a.q, (int32_t)a.k, a.scale);
}

template <class TI, class TO, int NT, int NV>
void go_causal_edge(const CausalSoftmaxArgs& a, hipStream_t s) {
    hipLaunchKernelGGL((sm_causal_edge<TI, TO, NT, NV>), dim3((unsigned)(a.batch * a.q)), dim3(NT), 0, s, a.x,
                       a.y, (int32_t)a.q, (int32_t)a.k, a.scale);
}

template <class TI, class TO>
kf_status run_causal(const CausalSoftmaxArgs& a, hipStream_t s, const char** variant) {
    if (a.batch * a.q > (int64_t)INT32_MAX || a.k > (int64_t)INT32_MAX || a.q > (int64_t)INT32_MAX) {
        set_error("softmax_causal: %lld rows of %lld exceed the grid limit", (long long)(a.batch * a.q),
                  (long long)a.k);
        return KF_ERR_UNSUPPORTED_LAYOUT;
    }
    const bool vec = (a.k % TI::vec == 0) && (a.k % TO::vec == 0) && ((uintptr_t)a.x % 16 == 0) &&
                     ((uintptr_t)a.y % 16 == 0);
    // Rows that are not whole vectors, on aligned bases: masked vectors
    // covering each row (at most ceil((k - 1) / VEC) + 1 of them).
    const bool edge = !vec && a.k >= TI::vec && ((uintptr_t)a.x % 16 == 0) && ((uintptr_t)a.y % 16 == 0);
    const int64_t slots = vec ? a.k / TI::vec : a.k;
    bool done = false;
    if (edge) {
        const int64_t eslots = (a.k - 1 + TI::vec - 1) / TI::vec + 1;
#define KF_CAUSAL_EDGE(NT, NV)                                                \
    if (!done && eslots <= (int64_t)(NT) * (NV)) {                            \
        go_causal_edge<TI, TO, NT, NV>(a, s);                                 \
        *variant = "sm_causal_edge_nt" #NT "_nv" #NV;                         \
        done = true;                                                          \
    }
        KF_CAUSAL_EDGE(64, 2)
        KF_CAUSAL_EDGE(128, 2)
        KF_CAUSAL_EDGE(128, 3)
        // Three waves of three slots for the 513 masked vectors of a 4097-key
        // bf16 row: 75.1 us against 78.4 us for 128 x 5 ([1, 8, 4097, 4097],
        // graph replays; the same cut on the non-causal rows, 320 x 2, was
        // slower than 256 x 3: 97.8 against 92.5 us).
        KF_CAUSAL_EDGE(192, 3)
        KF_CAUSAL_EDGE(128, 5)
        KF_CAUSAL_EDGE(512, 2)
        KF_CAUSAL_EDGE(512, 3)
        KF_CAUSAL_EDGE(1024, 2)
        KF_CAUSAL_EDGE(1024, 3)
        KF_CAUSAL_EDGE(1024, 5)
        if constexpr (TI::vec == 4) {
            KF_CAUSAL_EDGE(1024, 9)
        }
#undef KF_CAUSAL_EDGE
    }
#define KF_CAUSAL(NT, NV)                                                                                    \
    if (!done && slots <= (int64_t)(NT) * (NV)) {                                                            \
        if (vec) go_causal<TI, TO, NT, NV, true>(a, s);                                                      \
        else go_causal<TI, TO, NT, NV, false>(a, s);                                                         \
        *variant = vec ? "sm_causal_vec_nt" #NT "_nv" #NV : "sm_causal_scalar_nt" #NT "_nv" #NV;             \
        done = true;                                                                                         \
    }
    // 128 x 4 for rows of 2049-4096 keys: 67.1 us against 70.0 us for
    // 256 x 2 (and 67.3 for 64 x 8) on the causal attention workload (half
    // as many waves per row, so fewer of them sit idle on rows whose visible
    // prefix is short).  The unmasked softmax keeps 256 x 2 (87.4 against
    // 88.8 us for 128 x 4).
    KF_CAUSAL(64, 1)
    KF_CAUSAL(64, 2)
    KF_CAUSAL(128, 2)
    KF_CAUSAL(128, 4)
    KF_CAUSAL(512, 2)
    KF_CAUSAL(1024, 2)
    KF_CAUSAL(1024, 4)
    KF_CAUSAL(1024, 8)
#undef KF_CAUSAL
    if (!done) {
        // Beyond the register-resident tables: stream the row twice, with
        // 16-byte vectors wherever the bases are aligned.
        const dim3 g((unsigned)(a.batch * a.q)), b(1024);
        const int64_t total = a.batch * a.q * a.k;
        if (vec) {
            hipLaunchKernelGGL((sm_causal_stream<TI, TO, 1024, kStreamVec>), g, b, 0, s, a.x, a.y, a.q, a.k, a.scale,
                               total);
            *variant = "sm_causal_stream_vec";
        } else if (edge) {
            hipLaunchKernelGGL((sm_causal_stream<TI, TO, 1024, kStreamEdge>), g, b, 0, s, a.x, a.y, a.q, a.k, a.scale,
                               total);
            *variant = "sm_causal_stream_edge";
        } else {
            hipLaunchKernelGGL((sm_causal_stream<TI, TO, 1024, kStreamScalar>), g, b, 0, s, a.x, a.y, a.q, a.k,
                               a.scale, total);
            *variant = "sm_causal_stream_scalar";
        }
    }
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) {
        set_error("softmax_causal launch failed: %s", hipGetErrorString(err));
        return KF_ERR_HIP;
    }
    return KF_OK;
}


// --------------------------------------------------------------------------
// Split-row plan, from kernel-trace sweeps on MI355X (rows x lengths of
// bf16 scores with fp32 / bf16 output, cold HBM).  The exchange costs about
// 2.5 us over a workgroup-per-row launch, so a row is split only when
//   * the workgroup-per-row path would stream it twice (rows beyond the
//     register-resident kernels: more than 65536 elements, or 16384 when the
//     row is not whole 16-byte vectors), where splitting measured 2-7x
//     faster, or
//   * it moves at least 160 KiB (input plus output), from where splitting
//     measured 1.1-1.6x faster up to 64 rows;
// and only while the rows alone occupy fewer than kSplitMaxRows workgroups.
// Part size: the smallest (NV = 1, 2, 4, 8 16-byte vectors per thread, 4-32
// KiB of bf16) that leaves at most kSplitMaxParts parts per row: 16 KiB
// parts measured up to 1.5x faster than 4 KiB ones at 8-16 rows of 131072
// (64 parts per row is too many to gather), while for the decode step
// [1, 8, 1, 32768] 4 KiB parts (16 per row) beat 16 KiB ones, 4.95 against
// 5.41 us.  A larger NV halves the grid when rows x parts would exceed
// kSplitMaxGroups.
constexpr int64_t kSplitMaxRows = 128;
constexpr int64_t kSplitMaxGroups = 1024;
constexpr int64_t kSplitMaxParts = 16;
constexpr int64_t kSplitMinRowBytes = 160 << 10;

struct SplitPlan {
    int nv;         // 0: not split
    int64_t parts;
};

SplitPlan split_plan(const SoftmaxArgs& a) {
    SplitPlan none{0, 1};
    if (a.inner != 1 || a.outer >= kSplitMaxRows || a.outer < 1) return none;
    const int xvec = (a.xt == KF_FLOAT32) ? 4 : 8, yvec = (a.yt == KF_FLOAT32) ? 4 : 8;
    const int64_t row_bytes = a.len * (int64_t)((a.xt == KF_FLOAT32 ? 4 : 2) + (a.yt == KF_FLOAT32 ? 4 : 2));
    const bool whole_vectors = a.len % xvec == 0 && a.len % yvec == 0;
    const bool plain_streams = a.len > (whole_vectors ? 65536 : 16384);
    if (!plain_streams && row_bytes < kSplitMinRowBytes) return none;
    // Parts tile the row from the aligned boundary below its start: a row
    // not starting on one spans up to xvec - 1 more elements.
    const int64_t span = a.len + ((a.len % xvec) ? xvec - 1 : 0);
    for (int nv = 1; nv <= 8; nv *= 2) {
        const int64_t parts = (span + (int64_t)kSplitNT * nv * xvec - 1) / ((int64_t)kSplitNT * nv * xvec);
        if (parts < 2) return none;
        if (parts > kSplitMaxParts && nv < 8) continue;
        if (a.outer * parts <= kSplitMaxGroups) return SplitPlan{nv, parts};
    }
    return none;
}

uint32_t sm_wait_ticks() {
    static const uint32_t ticks = env_u32("KF355_SM_WAIT_TICKS", 10000u);
    return ticks;
}

template <class TI, class TO, int NV>
bool launch_split(const SoftmaxArgs& a, const SplitPlan& plan, void* workspace, hipStream_t s,
                  const char** variant) {
    const void* kernel = reinterpret_cast<const void*>(sm_split<TI, TO, NV>);
    static ResidencyCache capacity;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return false;
    const int64_t grid = a.outer * plan.parts;
    if ((int64_t)resident_capacity(capacity, dev, kernel, kSplitNT) < grid) return false;
    SplitParams p;
    p.x = a.x;
    p.y = a.y;
    p.ex = exchange_view(workspace, exchange_layout(a.outer, plan.parts), plan.parts, sm_wait_ticks());
    p.len = a.len;
    p.total = a.outer * a.len;
    hipLaunchKernelGGL((sm_split<TI, TO, NV>), dim3((unsigned)grid), dim3(kSplitNT), 0, s, p);
    *variant = NV == 1 ? "sm_split_nv1" : NV == 2 ? "sm_split_nv2" : NV == 4 ? "sm_split_nv4" : "sm_split_nv8";
    return true;
}

template <class TI, class TO>
kf_status run_split(const SoftmaxArgs& a, void* workspace, hipStream_t s, const char** variant) {
    const SplitPlan plan = split_plan(a);
    // In-place rows are not split (the recompute fallback re-reads x), nor
    // are buffers off a 16-byte boundary (the parts' vectors would not be).
    const bool ok = plan.nv != 0 && workspace && a.x != a.y && (uintptr_t)a.x % 16 == 0 &&
                    (uintptr_t)a.y % 16 == 0;
    bool launched = false;
    if (ok) {
        switch (plan.nv) {
            case 1: launched = launch_split<TI, TO, 1>(a, plan, workspace, s, variant); break;
            case 2: launched = launch_split<TI, TO, 2>(a, plan, workspace, s, variant); break;
            case 4: launched = launch_split<TI, TO, 4>(a, plan, workspace, s, variant); break;
            default: launched = launch_split<TI, TO, 8>(a, plan, workspace, s, variant); break;
        }
    }
    if (!launched) return run<TI, TO>(a, s, variant);
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) {
        set_error("softmax split launch failed: %s", hipGetErrorString(err));
        return KF_ERR_HIP;
    }
    return KF_OK;
}

}  // namespace

kf_status softmax_launch(const SoftmaxArgs& a, hipStream_t s, const char** variant) {
    if (a.xt == KF_FLOAT32 && a.yt == KF_FLOAT32) return run<F32, F32>(a, s, variant);
    if (a.xt == KF_BFLOAT16 && a.yt == KF_BFLOAT16) return run<BF16, BF16>(a, s, variant);
    if (a.xt == KF_BFLOAT16 && a.yt == KF_FLOAT32) return run<BF16, F32>(a, s, variant);
    if (a.xt == KF_FLOAT16 && a.yt == KF_FLOAT16) return run<F16, F16>(a, s, variant);
    if (a.xt == KF_FLOAT16 && a.yt == KF_FLOAT32) return run<F16, F32>(a, s, variant);
    set_error("softmax: unsupported dtype pair");
    return KF_ERR_BAD_DTYPE;
}

}  // namespace kf

namespace kf {
kf_status softmax_causal_launch(const CausalSoftmaxArgs& a, hipStream_t s, const char** variant) {
    if (a.xt == KF_FLOAT32 && a.yt == KF_FLOAT32) return run_causal<F32, F32>(a, s, variant);
    if (a.xt == KF_BFLOAT16 && a.yt == KF_BFLOAT16) return run_causal<BF16, BF16>(a, s, variant);
    if (a.xt == KF_BFLOAT16 && a.yt == KF_FLOAT32) return run_causal<BF16, F32>(a, s, variant);
    if (a.xt == KF_FLOAT16 && a.yt == KF_FLOAT16) return run_causal<F16, F16>(a, s, variant);
    if (a.xt == KF_FLOAT16 && a.yt == KF_FLOAT32) return run_causal<F16, F32>(a, s, variant);
    set_error("softmax_causal: unsupported dtype pair");
    return KF_ERR_BAD_DTYPE;
}
}  // namespace kf

namespace kf {
size_t softmax_split_workspace_bytes(const SoftmaxArgs& a) {
    const SplitPlan plan = split_plan(a);
    return plan.nv == 0 ? 0 : exchange_layout(a.outer, plan.parts).total;
}

kf_status softmax_split_launch(const SoftmaxArgs& a, void* workspace, hipStream_t s, const char** variant) {
    if (a.xt == KF_FLOAT32 && a.yt == KF_FLOAT32) return run_split<F32, F32>(a, workspace, s, variant);
    if (a.xt == KF_BFLOAT16 && a.yt == KF_BFLOAT16) return run_split<BF16, BF16>(a, workspace, s, variant);
    if (a.xt == KF_BFLOAT16 && a.yt == KF_FLOAT32) return run_split<BF16, F32>(a, workspace, s, variant);
    if (a.xt == KF_FLOAT16 && a.yt == KF_FLOAT16) return run_split<F16, F16>(a, workspace, s, variant);
    if (a.xt == KF_FLOAT16 && a.yt == KF_FLOAT32) return run_split<F16, F32>(a, workspace, s, variant);
    set_error("softmax: unsupported dtype pair");
    return KF_ERR_BAD_DTYPE;
}
}  // namespace kf
