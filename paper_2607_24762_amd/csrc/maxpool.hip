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
//   mp_tile    NCHW 3x3 windows at stride 2 without dilation (the ResNet
//              stem's pooling) on rows of whole 16-byte vectors: a thread
//              owns 16 bytes of consecutive outputs and folds its windows
//              from registers (vector loads, no LDS).
//   mp_direct  NCHW planes whose band tile does not fit in LDS: one thread
//              per output, window loads from global memory.
//   mp_nhwc    channels last: one thread per (output pixel, 16-byte vector
//              of channels), so every window load is coalesced along C and
//              overlapping windows re-read from cache.
#include <math.h>

#include <type_traits>

#include "kf_device.hpp"
#include "kf_internal.h"

namespace kf {
namespace {

constexpr int kNT = 256;
constexpr int kBandBytes = 16 << 10;  // LDS budget of one band tile
constexpr int64_t kBandGroups = 2048;  // persistent band workgroups (8 per CU)
// mp_tile: output rows per thread.  On the ResNet stem one row (25.1 us)
// beats reusing the shared input row across two (27.4 us) or four (30.4 us):
// the extra threads keep more loads in flight, and the shared row comes
// from L2.
constexpr int kTileRows = 1;

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

// The running choice of one window, with its position (indices wanted).
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
    // The same step without branches, skipped where !valid: callers read
    // every window position (from a clamped address) before folding, so
    // the reads issue together instead of one branch and one wait each.
    __device__ __forceinline__ void consider_if(bool valid, uint32_t raw, int32_t pos) {
        // Bitwise, not short-circuit, operators: the compiler keeps this
        // as compares and selects instead of branching around each term.
        const float v = Raw<T>::value(raw);
        const bool first = valid & (at < 0);
        const bool take = valid & ((v > best) | (v != v));
        best = take ? v : best;
        bits = take ? raw : bits;
        at = (take | first) ? pos : at;
    }
    __device__ __forceinline__ uint32_t result() const { return bits; }
    __device__ __forceinline__ int32_t index() const { return at; }
};

// Canonical quiet NaN of each storage format.
template <class T>
constexpr uint32_t kQuietNaN = 0x7fc00000u;
template <>
constexpr uint32_t kQuietNaN<BF16> = 0x7fc0u;
template <>
constexpr uint32_t kQuietNaN<F16> = 0x7e00u;

// Storage bits of a float that holds a value of T exactly.
template <class T>
__device__ __forceinline__ uint32_t raw_of(float f) {
    if constexpr (std::is_same_v<T, F32>) return __float_as_uint(f);
    else if constexpr (std::is_same_v<T, BF16>) return __float_as_uint(f) >> 16;
    else return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)f);
}

// IEEE 754-2019 maximum of three (NaN propagates, -0 < +0): one
// v_maximum3_f32 on gfx950.
__device__ __forceinline__ float maximum3(float a, float b, float c) {
    return __builtin_elementwise_maximum(__builtin_elementwise_maximum(a, b), c);
}

// The value-only choice (no indices wanted): the window's maximum and
// whether it held a NaN.  Every element of a window converts to float
// exactly, so the maximum converts back exactly; a NaN window yields the
// canonical quiet NaN, and where +0 and -0 tie the result may be +0 (the
// two compare equal).  Two instructions per element instead of Pick's
// compare-and-select chain.
template <class T>
struct MaxOnly {
    float best = -INFINITY;
    bool nan = false;
    __device__ __forceinline__ void consider(uint32_t raw, int32_t) {
        const float v = Raw<T>::value(raw);
        best = fmaxf(best, v);
        nan = nan | (v != v);
    }
    __device__ __forceinline__ void consider_if(bool valid, uint32_t raw, int32_t) {
        const float v = Raw<T>::value(raw);
        best = valid ? fmaxf(best, v) : best;
        nan = nan | (valid & (v != v));
    }
    __device__ __forceinline__ uint32_t result() const { return nan ? kQuietNaN<T> : raw_of<T>(best); }
    __device__ __forceinline__ int32_t index() const { return -1; }
};

template <class T>
__device__ __forceinline__ MaxOnly<T> merge(const MaxOnly<T>& a, const MaxOnly<T>& b) {
    MaxOnly<T> m;
    m.best = fmaxf(a.best, b.best);
    m.nan = a.nan | b.nan;
    return m;
}

// Selection rule of a kernel: with indices the position-tracking Pick, else
// the value-only maximum.
template <class T, bool IDX>
using Select = std::conditional_t<IDX, Pick<T>, MaxOnly<T>>;

// Merge of two picks over consecutive stretches of the row-major scan (a
// before b): scanning b's elements after a's moves to b's pick exactly when
// b holds a greater element or a NaN, so the merged pick equals the pick of
// the whole scan; an empty a (no in-plane position yet) takes b.
// (Selected field by field: a select of whole structs would make the
// compiler keep them in scratch memory.)
template <class T>
__device__ __forceinline__ Pick<T> merge(const Pick<T>& a, const Pick<T>& b) {
    const bool take = (a.at < 0) | (b.best > a.best) | (b.best != b.best);
    Pick<T> m;
    m.best = take ? b.best : a.best;
    m.bits = take ? b.bits : a.bits;
    m.at = take ? b.at : a.at;
    return m;
}

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
// NCHW, bands of output rows, input rows in LDS.  Work item = (plane, band);
// a persistent workgroup walks items blockIdx.x, + gridDim.x, ...  In the
// vector form the next item's input span is loaded into registers while the
// current one is scanned from LDS and written, so every workgroup keeps
// loads in flight through its compute and store phases.

// Rows and span of one work item.
struct Band {
    int64_t plane;
    int o0, o1, r_lo, n;  // output rows [o0, o1), first input row, span elements
};
__device__ __forceinline__ Band band_of(const MPParams& p, int64_t item) {
    Band b;
    b.plane = item / p.bands;
    const int band = (int)(item - b.plane * p.bands);
    b.o0 = band * p.band_rows;
    b.o1 = min(p.oh, b.o0 + p.band_rows);
    b.r_lo = max(0, b.o0 * p.sh - p.ph);
    const int r_hi = min(p.h, (b.o1 - 1) * p.sh - p.ph + (p.kh - 1) * p.dh + 1);
    b.n = max(0, r_hi - b.r_lo) * p.w;
    return b;
}

template <class R>
__device__ __forceinline__ const R* band_src(const MPParams& p, const Band& b) {
    return static_cast<const R*>(p.x) + b.plane * p.h * p.w + (int64_t)b.r_lo * p.w;
}

// Scan the band's windows from LDS and write its outputs.  K > 0: a K x K
// window known at compile time, so the loops unroll and the K*K LDS reads
// of an output issue together.
template <class T, int K, bool IDX, class R>
__device__ __forceinline__ void band_outputs(const MPParams& p, const Band& b, const R* tile) {
    const int outs = (b.o1 - b.o0) * p.ow;
    R* dst = static_cast<R*>(p.y) + b.plane * p.oh * p.ow + (int64_t)b.o0 * p.ow;
    int64_t* idx = p.idx ? p.idx + b.plane * p.oh * p.ow + (int64_t)b.o0 * p.ow : nullptr;
    // Output q of the band is (o0 + q / ow, q % ow); the quotient is kept
    // incrementally (q grows by kNT per step) instead of dividing.
    int i = b.o0 + (int)threadIdx.x / p.ow, j = (int)threadIdx.x - ((int)threadIdx.x / p.ow) * p.ow;
    const int di = kNT / p.ow, dj = kNT - di * p.ow;
    for (int q = threadIdx.x; q < outs; q += kNT) {
        Select<T, IDX> pk;
        // Positions outside the plane read the tile's first element and
        // are skipped (the tile always holds at least one row).
        auto at = [&](int a, int c) {
            const int r = i * p.sh - p.ph + a * p.dh;
            const int col = j * p.sw - p.pw + c * p.dw;
            const bool ok = r >= 0 && r < p.h && col >= 0 && col < p.w;
            pk.consider_if(ok, tile[ok ? (r - b.r_lo) * p.w + col : 0], r * p.w + col);
        };
        if constexpr (K > 0) {
#pragma unroll
            for (int a = 0; a < K; ++a)
#pragma unroll
                for (int c = 0; c < K; ++c) at(a, c);
        } else {
            for (int a = 0; a < p.kh; ++a)
                for (int c = 0; c < p.kw; ++c) at(a, c);
        }
        __builtin_nontemporal_store((R)pk.result(), dst + q);
        if constexpr (IDX) __builtin_nontemporal_store((int64_t)pk.index(), idx + q);
        i += di;
        j += dj;
        if (j >= p.ow) {
            j -= p.ow;
            ++i;
        }
    }
}

// K x K window, stride S in both directions, no dilation: each thread owns a
// vertical strip of up to kStripRows outputs in one column.  Its K column
// positions (and whether they are in the plane) are fixed; each input row
// is reduced to a row pick once, and output i + 1 reuses the K - S row
// picks it shares with output i.
constexpr int kStripRows = 4;

// Position of column c inside a staged row: identity, or for stride-2
// scans the row split into its even columns then its odd columns, so that
// lanes reading columns 2j-1, 2j, 2j+1 for consecutive j hit consecutive
// LDS words (no bank conflicts).
template <int S>
__device__ __forceinline__ int tile_col(int c, int half) {
    if constexpr (S == 2) return (c & 1) ? half + (c >> 1) : (c >> 1);
    else return c;
}

template <class T, int K, int S, bool IDX, class R>
__device__ __forceinline__ void band_outputs_strip(const MPParams& p, const Band& b, const R* tile) {
    const int half = (p.w + 1) >> 1;
    const int rows = b.o1 - b.o0;
    const int runs = (rows + kStripRows - 1) / kStripRows;
    const int tasks = runs * p.ow;
    R* dst = static_cast<R*>(p.y) + b.plane * p.oh * p.ow;
    int64_t* idx = p.idx ? p.idx + b.plane * p.oh * p.ow : nullptr;
    for (int t = threadIdx.x; t < tasks; t += kNT) {
        const int run = t / p.ow, j = t - run * p.ow;
        const int i0 = b.o0 + run * kStripRows, i1 = min(b.o1, i0 + kStripRows);
        int col[K], tcol[K];
        bool col_ok[K];
#pragma unroll
        for (int c = 0; c < K; ++c) {
            col[c] = j * S - p.pw + c;
            col_ok[c] = col[c] >= 0 && col[c] < p.w;
            tcol[c] = tile_col<S>(col_ok[c] ? col[c] : 0, half);  // outside: any in-tile column
        }
        // All K reads of a row issue before the fold (rows outside the
        // plane read the tile's first row and are skipped).
        auto row_pick = [&](int r) {
            Select<T, IDX> pk;
            const bool r_ok = r >= 0 && r < p.h;
            const R* row = tile + (r_ok ? r - b.r_lo : 0) * p.w;
            uint32_t raw[K];
#pragma unroll
            for (int c = 0; c < K; ++c) raw[c] = row[tcol[c]];
#pragma unroll
            for (int c = 0; c < K; ++c) pk.consider_if(r_ok && col_ok[c], raw[c], r * p.w + col[c]);
            return pk;
        };
        Select<T, IDX> rp[K];  // row picks of the current output's K rows
#pragma unroll
        for (int a = 0; a < K; ++a) rp[a] = row_pick(i0 * S - p.ph + a);
        for (int i = i0; i < i1; ++i) {
            if (i > i0) {
                if constexpr (S < K) {
#pragma unroll
                    for (int a = 0; a < K - S; ++a) rp[a] = rp[a + S];
#pragma unroll
                    for (int a = K - S; a < K; ++a) rp[a] = row_pick(i * S - p.ph + a);
                } else {
#pragma unroll
                    for (int a = 0; a < K; ++a) rp[a] = row_pick(i * S - p.ph + a);
                }
            }
            Select<T, IDX> pk = rp[0];
#pragma unroll
            for (int a = 1; a < K; ++a) pk = merge(pk, rp[a]);
            const int64_t o = (int64_t)i * p.ow + j;
            __builtin_nontemporal_store((R)pk.result(), dst + o);
            if constexpr (IDX) __builtin_nontemporal_store((int64_t)pk.index(), idx + o);
        }
    }
}

// Vector staging: the span starts on a 16-byte boundary (w and h*w are
// whole vectors, the base is aligned) and is whole vectors; at most
// kBandBytes, so kStageVecs 16-byte vectors per thread.
constexpr int kStageVecs = kBandBytes / 16 / kNT;

template <class R>
__device__ __forceinline__ void stage_load(const MPParams& p, const Band& b, u32x4 (&r)[kStageVecs]) {
    const u32x4* s4 = reinterpret_cast<const u32x4*>(band_src<R>(p, b));
    const int nv = b.n / (16 / (int)sizeof(R));
#pragma unroll
    for (int d = 0; d < kStageVecs; ++d) {
        const int v = threadIdx.x + d * kNT;
        r[d] = s4[v < nv ? v : 0];
    }
}

// Writes the staged vectors into the tile; for S == 2 each row is split
// into even then odd columns (see tile_col): a vector starts on an even
// column (w is whole vectors), so its even and odd halves land as two
// contiguous runs of VEC/2 elements.
template <class R, int S>
__device__ __forceinline__ void stage_store(const MPParams& p, const Band& b, const u32x4 (&r)[kStageVecs],
                                            u32x4* lds) {
    constexpr int VEC = 16 / (int)sizeof(R);
    const int nv = b.n / VEC;
    const int half = p.w >> 1;
#pragma unroll
    for (int d = 0; d < kStageVecs; ++d) {
        const int v = threadIdx.x + d * kNT;
        if (v < nv) {
            if constexpr (S == 2) {
                // Each half is 8 bytes: packed into one 64-bit word and
                // written with one 8-byte-aligned LDS store (c0 / 2 is a
                // multiple of VEC / 2, and w / 2 * sizeof(R) of 8).
                const Lanes<R, VEC> in = __builtin_bit_cast(Lanes<R, VEC>, r[d]);
                uint64_t ev = 0, od = 0;
#pragma unroll
                for (int k = 0; k < VEC / 2; ++k) {
                    ev |= (uint64_t)in.v[2 * k] << (k * 8 * sizeof(R));
                    od |= (uint64_t)in.v[2 * k + 1] << (k * 8 * sizeof(R));
                }
                const int e = v * VEC, rr = e / p.w, c0 = e - rr * p.w;
                R* row = reinterpret_cast<R*>(lds) + rr * p.w;
                *reinterpret_cast<uint64_t*>(row + (c0 >> 1)) = ev;
                *reinterpret_cast<uint64_t*>(row + half + (c0 >> 1)) = od;
            } else {
                lds[v] = r[d];
            }
        }
    }
}

// S > 0: the strip form above (K x K, stride S, no dilation).
template <class T, int K, int S, bool IDX, class R>
__device__ __forceinline__ void band_scan(const MPParams& p, const Band& b, const R* tile) {
    if constexpr (S > 0) band_outputs_strip<T, K, S, IDX>(p, b, tile);
    else band_outputs<T, K, IDX>(p, b, tile);
}

template <class T, bool VECTOR, int K, int S, bool IDX>
__global__ __launch_bounds__(kNT) void mp_band(MPParams p) {
    using R = typename Raw<T>::type;
    extern __shared__ u32x4 lds_vec[];
    R* tile = reinterpret_cast<R*>(lds_vec);
    const int64_t items = p.planes * p.bands;
    int64_t item = blockIdx.x;
    if (item >= items) return;
    Band b = band_of(p, item);
    if constexpr (VECTOR) {
        u32x4 r[kStageVecs];
        stage_load<R>(p, b, r);
        while (true) {
            stage_store<R, S>(p, b, r, lds_vec);
            __syncthreads();
            const int64_t next = item + gridDim.x;
            Band nb = b;
            if (next < items) {
                nb = band_of(p, next);
                stage_load<R>(p, nb, r);  // in flight while this band is scanned
            }
            band_scan<T, K, S, IDX>(p, b, tile);
            if (next >= items) break;
            __syncthreads();  // the tile is rewritten next
            item = next;
            b = nb;
        }
    } else {
        while (true) {
            const R* src = band_src<R>(p, b);
            const int half = (p.w + 1) >> 1;
            for (int e = threadIdx.x; e < b.n; e += kNT) {
                const int rr = e / p.w, c = e - rr * p.w;
                tile[rr * p.w + tile_col<S>(c, half)] = src[e];
            }
            __syncthreads();
            band_scan<T, K, S, IDX>(p, b, tile);
            item += gridDim.x;
            if (item >= items) break;
            __syncthreads();
            b = band_of(p, item);
        }
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
// Workgroups go to the 8 XCDs in turn (dispatch order L goes to XCD L % 8).
// xcd_contiguous renumbers them so that XCD x runs one contiguous range of
// the T logical tiles: x gets q = T / 8 tiles, one more when x < T % 8, and
// starts at x * q + min(x, T % 8).  A bijection on [0, T).
__device__ __forceinline__ uint32_t xcd_contiguous(uint32_t L, uint32_t T) {
    const uint32_t q = T >> 3, r = T & 7, x = L & 7;
    return x * q + min(x, r) + (L >> 3);
}

// NHWC: thread per (output pixel, VEC channels).  VEC = 16 bytes of
// channels when c is whole vectors and the bases are aligned, else 1.  The
// grid is (tiles per sample, samples), renumbered with xcd_contiguous, so
// tiles of neighbouring output rows, whose windows share input rows, run on
// one XCD and find those rows in its L2 (in dispatch order they would land
// on different XCDs and each fetch the shared rows again).  Inside a sample
// every index fits 32 bits (checked on the host), so the index arithmetic
// is 32-bit.
template <class T, int VEC, int K, bool IDX>
__global__ __launch_bounds__(kNT) void mp_nhwc(MPParams p) {
    using R = typename Raw<T>::type;
    const uint32_t tiles = gridDim.x;
    const uint32_t logical = xcd_contiguous(blockIdx.y * tiles + blockIdx.x, tiles * gridDim.y);
    const uint32_t sample = logical / tiles;
    const uint32_t cvs = (uint32_t)p.c / VEC;
    const uint32_t t = (logical - sample * tiles) * kNT + threadIdx.x;
    if (t >= (uint32_t)p.oh * (uint32_t)p.ow * cvs) return;
    const uint32_t pix = t / cvs;
    const int cv = (int)(t - pix * cvs);
    const int i = (int)(pix / (uint32_t)p.ow);
    const int j = (int)(pix - (uint32_t)i * (uint32_t)p.ow);
    const int64_t nn = sample;
    const R* xs = static_cast<const R*>(p.x);
    Select<T, IDX> pk[VEC];
    auto load = [&](int r, int col) {
        const int64_t e = ((nn * p.h + r) * p.w + col) * p.c + (int64_t)cv * VEC;
        Lanes<R, VEC> v;
        if constexpr (VEC == 1) v.v[0] = xs[e];
        else v = __builtin_bit_cast(Lanes<R, VEC>, *reinterpret_cast<const u32x4*>(xs + e));
        return v;
    };
    if constexpr (K > 0) {
        // Every window position is loaded first (positions outside the
        // plane from a clamped in-plane address, then skipped), so all K*K
        // loads are in flight together.
        Lanes<R, VEC> v[K * K];
#pragma unroll
        for (int a = 0; a < K; ++a)
#pragma unroll
            for (int c = 0; c < K; ++c) {
                const int r = min(max(i * p.sh - p.ph + a * p.dh, 0), p.h - 1);
                const int col = min(max(j * p.sw - p.pw + c * p.dw, 0), p.w - 1);
                v[a * K + c] = load(r, col);
            }
#pragma unroll
        for (int a = 0; a < K; ++a)
#pragma unroll
            for (int c = 0; c < K; ++c) {
                const int r = i * p.sh - p.ph + a * p.dh;
                const int col = j * p.sw - p.pw + c * p.dw;
                const bool ok = r >= 0 && r < p.h && col >= 0 && col < p.w;
#pragma unroll
                for (int k = 0; k < VEC; ++k) pk[k].consider_if(ok, v[a * K + c].v[k], r * p.w + col);
            }
    } else {
        for (int a = 0; a < p.kh; ++a) {
            const int r = i * p.sh - p.ph + a * p.dh;
            if (r < 0 || r >= p.h) continue;
            for (int c = 0; c < p.kw; ++c) {
                const int col = j * p.sw - p.pw + c * p.dw;
                if (col < 0 || col >= p.w) continue;
                const Lanes<R, VEC> v = load(r, col);
#pragma unroll
                for (int k = 0; k < VEC; ++k) pk[k].consider(v.v[k], r * p.w + col);
            }
        }
    }
    const int64_t o = (nn * p.oh * p.ow + pix) * p.c + (int64_t)cv * VEC;
    Lanes<R, VEC> out;
#pragma unroll
    for (int k = 0; k < VEC; ++k) out.v[k] = (R)pk[k].result();
    if constexpr (VEC == 1) {
        __builtin_nontemporal_store(out.v[0], static_cast<R*>(p.y) + o);
    } else {
        __builtin_nontemporal_store(__builtin_bit_cast(u32x4, out), reinterpret_cast<u32x4*>(static_cast<R*>(p.y) + o));
    }
    if constexpr (IDX) {
#pragma unroll
        for (int k = 0; k < VEC; ++k) __builtin_nontemporal_store((int64_t)pk[k].index(), p.idx + o + k);
    }
}

// --------------------------------------------------------------------------
// NCHW 3x3 windows, stride 2, no dilation, padding PW = 0 or 1 across (any
// padding down): the ResNet stem's pooling, on planes whose rows are whole
// 16-byte vectors.  A thread owns E = 16 / sizeof(T) consecutive outputs in
// each of ROWS consecutive output rows of one plane.  Its windows span
// 2 * ROWS + 1 input rows and 2E + 1 columns: per row two 16-byte vectors
// (columns 2 * j0 .. 2 * j0 + 2E - 1) and one halo element (the column to
// the left with padding 1, to the right without), all loaded before any
// folding, from clamped addresses where a row or column lies outside the
// plane.  Each input row is folded into E row picks (three columns per
// output), and output rows that share an input row reuse its picks, so no
// element is read twice from registers or memory by one thread.  Lanes run
// along an output row, so a wave's vector loads cover input rows
// contiguously; workgroups are numbered XCD-contiguously, so neighbouring
// row groups, which share one input row, run on one XCD.  No LDS, no
// barrier.
//
// EXACT (value only, no indices; the host sets it when no vector column
// lies right of the plane, 2 * E * ceil(ow / E) <= w): then every clamped
// load is a duplicate of an element of the same window (a window is an
// interval of rows and of columns that meets the plane, and clamping moves
// an outside row or column to the nearest one inside), which cannot change
// a maximum, so the folds need no masks: one maximum3 per output per row
// and one across rows.  Such a NaN result is a quiet NaN (an input NaN's
// payload, quieted), not necessarily the canonical one.
template <class T, bool IDX, int ROWS, int PW, bool EXACT>
__global__ __launch_bounds__(kNT) void mp_tile(MPParams p) {
    static_assert(!(IDX && EXACT), "positions need the masked fold");
    using R = typename Raw<T>::type;
    constexpr int E = 16 / sizeof(R);
    constexpr int IN = 2 * ROWS + 1;  // input rows under a thread's windows
    constexpr int COLS = 2 * E + 1;   // input columns under them
    const uint32_t gw = ((uint32_t)p.ow + E - 1) / E;        // column groups per output row
    const uint32_t rg = ((uint32_t)p.oh + ROWS - 1) / ROWS;  // row groups per plane
    const uint32_t t = xcd_contiguous(blockIdx.x, gridDim.x) * kNT + threadIdx.x;
    if (t >= (uint32_t)p.planes * rg * gw) return;  // the host keeps this product below 2^31
    const uint32_t g = t % gw;
    const uint32_t rest = t / gw;
    const uint32_t plane = rest / rg;
    const int i0 = (int)(rest - plane * rg) * ROWS;  // first output row
    const int j0 = (int)g * E;                       // first output column
    const int c0 = 2 * j0 - PW;                      // column of value 0 below
    const int r0 = 2 * i0 - p.ph;                    // input row of row 0 below
    const R* xp = static_cast<const R*>(p.x) + (int64_t)plane * p.h * p.w;

    // v[a][m]: input row r0 + a, column c0 + m.  With PW = 1 the halo is
    // m = 0 and the vectors m = 1 .. 2E; with PW = 0 the vectors are
    // m = 0 .. 2E - 1 and the halo m = 2E.  A vector starts at a multiple
    // of E, so it lies wholly inside or wholly outside the row (w % E == 0).
    R v[IN][COLS];
    const int va = 2 * j0, vb = 2 * j0 + E, hc = PW ? 2 * j0 - 1 : 2 * j0 + 2 * E;
    const int va_c = min(va, p.w - E), vb_c = min(vb, p.w - E), hc_c = min(max(hc, 0), p.w - 1);
    const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
    for (int a = 0; a < IN; ++a) {
        const R* row = xp + (int64_t)min(max(r0 + a, 0), p.h - 1) * p.w;
        const Lanes<R, E> A = __builtin_bit_cast(Lanes<R, E>, *reinterpret_cast<const u32x4*>(row + va_c));
        const Lanes<R, E> B = __builtin_bit_cast(Lanes<R, E>, *reinterpret_cast<const u32x4*>(row + vb_c));
#pragma unroll
        for (int k = 0; k < E; ++k) {
            v[a][PW + k] = A.v[k];
            v[a][PW + E + k] = B.v[k];
        }
        if constexpr (EXACT && PW == 1) {
            // The left halo (column 2 * j0 - 1) is the last element of the
            // previous lane's B when that lane holds the previous column
            // group of the same output row (g > 0): a DPP wave shift by one
            // lane instead of a load.  Lane 0 of the wave, which has no
            // previous lane, loads it (the shift hands lane 0 its own
            // operand); g == 0 has the halo in the padding, clamped to
            // column 0, which A already holds (a duplicate, harmless to a
            // maximum).  Measured 25.1 -> 24.4 us on the ResNet stem.
            uint32_t own = 0;
            if (lane == 0) own = (uint32_t)row[hc_c];
            const uint32_t prev = (uint32_t)__builtin_amdgcn_update_dpp((int)own, (int)(uint32_t)B.v[E - 1],
                                                                        0x138 /* wave_shr:1 */, 0xF, 0xF, false);
            v[a][0] = g == 0 ? A.v[0] : (R)prev;
        } else {
            v[a][PW ? 0 : 2 * E] = row[hc_c];
        }
    }

    Lanes<R, E> out[ROWS];
    int32_t at[ROWS][E];
    if constexpr (EXACT) {
        float hm[IN][E];  // row maxima of each output's three columns
#pragma unroll
        for (int a = 0; a < IN; ++a)
#pragma unroll
            for (int k = 0; k < E; ++k)
                hm[a][k] = maximum3(Raw<T>::value(v[a][2 * k]), Raw<T>::value(v[a][2 * k + 1]),
                                    Raw<T>::value(v[a][2 * k + 2]));
#pragma unroll
        for (int q = 0; q < ROWS; ++q)
#pragma unroll
            for (int k = 0; k < E; ++k)
                out[q].v[k] = (R)raw_of<T>(maximum3(hm[2 * q][k], hm[2 * q + 1][k], hm[2 * q + 2][k]));
    } else {
        // Row picks: rp[a][k] folds columns 2k, 2k + 1, 2k + 2 of row a, in
        // order, skipping positions outside the plane.
        Select<T, IDX> rp[IN][E];
#pragma unroll
        for (int a = 0; a < IN; ++a) {
            const int r = r0 + a;
            const bool row_ok = (r >= 0) & (r < p.h);
#pragma unroll
            for (int k = 0; k < E; ++k)
#pragma unroll
                for (int m = 2 * k; m < 2 * k + 3; ++m) {
                    const int col = c0 + m;
                    rp[a][k].consider_if(row_ok & (col >= 0) & (col < p.w), v[a][m], r * p.w + col);
                }
        }
#pragma unroll
        for (int q = 0; q < ROWS; ++q)
#pragma unroll
            for (int k = 0; k < E; ++k) {
                const Select<T, IDX> s = merge(merge(rp[2 * q][k], rp[2 * q + 1][k]), rp[2 * q + 2][k]);
                out[q].v[k] = (R)s.result();
                at[q][k] = s.index();
            }
    }

    R* yp = static_cast<R*>(p.y) + (int64_t)plane * p.oh * p.ow;
    const bool whole = (p.ow % E == 0);  // output rows are whole 16-byte vectors
#pragma unroll
    for (int q = 0; q < ROWS; ++q) {
        const int i = i0 + q;
        if (i >= p.oh) break;
        const int64_t o = (int64_t)i * p.ow + j0;
        if (whole) {
            __builtin_nontemporal_store(__builtin_bit_cast(u32x4, out[q]), reinterpret_cast<u32x4*>(yp + o));
        } else {
#pragma unroll
            for (int k = 0; k < E; ++k)
                if (j0 + k < p.ow) yp[o + k] = out[q].v[k];
        }
        if constexpr (IDX) {
            // A lane's E indices are 8E contiguous bytes: written as 16-byte
            // stores that the cache merges into whole lines with the
            // neighbouring lanes' (8-byte non-temporal stores at a 32-byte
            // lane stride measured 2.3x slower).
            int64_t* ip = p.idx + (int64_t)plane * p.oh * p.ow + o;
            if (whole) {
#pragma unroll
                for (int k = 0; k < E; k += 2) {
                    const u32x4 pair = {(uint32_t)at[q][k], at[q][k] < 0 ? ~0u : 0u, (uint32_t)at[q][k + 1],
                                        at[q][k + 1] < 0 ? ~0u : 0u};
                    *reinterpret_cast<u32x4*>(ip + k) = pair;
                }
            } else {
#pragma unroll
                for (int k = 0; k < E; ++k)
                    if (j0 + k < p.ow) ip[k] = at[q][k];
            }
        }
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
        const int64_t per_sample = a.oh * a.ow * (vec ? a.c / VEC : a.c);
        const int64_t tiles = (per_sample + kNT - 1) / kNT;
        if (per_sample > INT32_MAX || a.n > 65535 || tiles * a.n > (int64_t)UINT32_MAX) {
            set_error("max_pool2d: %lld threads per sample or %lld samples exceed the channels-last grid",
                      (long long)per_sample, (long long)a.n);
            return KF_ERR_UNSUPPORTED_LAYOUT;
        }
        const dim3 grid((unsigned)tiles, (unsigned)a.n);
        const int k = (a.kh == a.kw && (a.kh == 2 || a.kh == 3)) ? a.kh : 0;
        auto go = [&](auto kernel) { hipLaunchKernelGGL(kernel, grid, dim3(kNT), 0, s, p); };
        auto pick = [&](auto idx_tag) {
            constexpr bool I = decltype(idx_tag)::value;
            if (vec) {
                if (k == 3) go(mp_nhwc<T, VEC, 3, I>);
                else if (k == 2) go(mp_nhwc<T, VEC, 2, I>);
                else go(mp_nhwc<T, VEC, 0, I>);
            } else {
                if (k == 3) go(mp_nhwc<T, 1, 3, I>);
                else if (k == 2) go(mp_nhwc<T, 1, 2, I>);
                else go(mp_nhwc<T, 1, 0, I>);
            }
        };
        if (a.idx) pick(std::true_type{});
        else pick(std::false_type{});
        static const char* names[2][2][3] = {
            {{"mp_nhwc_scalar", "mp_nhwc_scalar_k2", "mp_nhwc_scalar_k3"},
             {"mp_nhwc_vec", "mp_nhwc_vec_k2", "mp_nhwc_vec_k3"}},
            {{"mp_nhwc_scalar_idx", "mp_nhwc_scalar_k2_idx", "mp_nhwc_scalar_k3_idx"},
             {"mp_nhwc_vec_idx", "mp_nhwc_vec_k2_idx", "mp_nhwc_vec_k3_idx"}}};
        *variant = names[a.idx ? 1 : 0][vec ? 1 : 0][k == 0 ? 0 : k - 1];
    } else if (a.kh == 3 && a.kw == 3 && a.sh == 2 && a.sw == 2 && a.dh == 1 && a.dw == 1 && a.w % VEC == 0 &&
               (uintptr_t)a.x % 16 == 0 && (uintptr_t)a.y % 16 == 0 && (uintptr_t)a.idx % 16 == 0 &&
               p.planes * ((a.oh + kTileRows - 1) / kTileRows) * ((a.ow + VEC - 1) / VEC) < INT32_MAX) {
        const int64_t threads = p.planes * ((a.oh + kTileRows - 1) / kTileRows) * ((a.ow + VEC - 1) / VEC);
        const dim3 grid((unsigned)((threads + kNT - 1) / kNT));
        auto go = [&](auto kernel) { hipLaunchKernelGGL(kernel, grid, dim3(kNT), 0, s, p); };
        const bool exact = 2 * VEC * ((a.ow + VEC - 1) / VEC) <= a.w;
        if (a.idx) {
            if (a.pw) go(mp_tile<T, true, kTileRows, 1, false>);
            else go(mp_tile<T, true, kTileRows, 0, false>);
            *variant = "mp_tile_idx";
        } else if (exact) {
            if (a.pw) go(mp_tile<T, false, kTileRows, 1, true>);
            else go(mp_tile<T, false, kTileRows, 0, true>);
            *variant = "mp_tile_exact";
        } else {
            if (a.pw) go(mp_tile<T, false, kTileRows, 1, false>);
            else go(mp_tile<T, false, kTileRows, 0, false>);
            *variant = "mp_tile";
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
            // Persistent workgroups: enough to fill every CU several times
            // over (each walks items with stride gridDim.x).
            const int64_t items = p.planes * bands;
            const int64_t grid = items < kBandGroups ? items : kBandGroups;
            const int64_t in_rows = (br - 1) * a.sh + eff;
            const size_t lds = (size_t)(((in_rows * row_bytes) + 15) / 16 * 16);
            const bool vec = a.w % VEC == 0 && (a.h * a.w) % VEC == 0 && (uintptr_t)a.x % 16 == 0;
            // Compile-time forms: square 3x3 / 2x2 windows (unrolled scan);
            // with equal strides 1 or 2 and no dilation, the strip scan.
            const int k = (a.kh == a.kw && (a.kh == 2 || a.kh == 3)) ? a.kh : 0;
            const bool strip = k != 0 && a.sh == a.sw && a.dh == 1 && a.dw == 1 &&
                               ((k == 3 && (a.sh == 1 || a.sh == 2)) || (k == 2 && a.sh == 2));
            const int sv = strip ? a.sh : 0;
            auto go = [&](auto kernel) { hipLaunchKernelGGL(kernel, dim3((unsigned)grid), dim3(kNT), lds, s, p); };
            auto pick = [&](auto vec_tag, auto idx_tag) {
                constexpr bool V = decltype(vec_tag)::value, I = decltype(idx_tag)::value;
                if (k == 3 && sv == 2) go(mp_band<T, V, 3, 2, I>);
                else if (k == 3 && sv == 1) go(mp_band<T, V, 3, 1, I>);
                else if (k == 2 && sv == 2) go(mp_band<T, V, 2, 2, I>);
                else if (k == 3) go(mp_band<T, V, 3, 0, I>);
                else if (k == 2) go(mp_band<T, V, 2, 0, I>);
                else go(mp_band<T, V, 0, 0, I>);
            };
            auto with_idx = [&](auto vec_tag) {
                if (a.idx) pick(vec_tag, std::true_type{});
                else pick(vec_tag, std::false_type{});
            };
            if (vec) with_idx(std::true_type{});
            else with_idx(std::false_type{});
            static const char* names[2][2][3][3] = {
                {{{"mp_band_scalar", "mp_band_scalar", "mp_band_scalar"},
                  {"mp_band_scalar_k2", "mp_band_scalar_k2", "mp_band_scalar_k2_strip_s2"},
                  {"mp_band_scalar_k3", "mp_band_scalar_k3_strip_s1", "mp_band_scalar_k3_strip_s2"}},
                 {{"mp_band_vec", "mp_band_vec", "mp_band_vec"},
                  {"mp_band_vec_k2", "mp_band_vec_k2", "mp_band_vec_k2_strip_s2"},
                  {"mp_band_vec_k3", "mp_band_vec_k3_strip_s1", "mp_band_vec_k3_strip_s2"}}},
                {{{"mp_band_scalar_idx", "mp_band_scalar_idx", "mp_band_scalar_idx"},
                  {"mp_band_scalar_k2_idx", "mp_band_scalar_k2_idx", "mp_band_scalar_k2_strip_s2_idx"},
                  {"mp_band_scalar_k3_idx", "mp_band_scalar_k3_strip_s1_idx", "mp_band_scalar_k3_strip_s2_idx"}},
                 {{"mp_band_vec_idx", "mp_band_vec_idx", "mp_band_vec_idx"},
                  {"mp_band_vec_k2_idx", "mp_band_vec_k2_idx", "mp_band_vec_k2_strip_s2_idx"},
                  {"mp_band_vec_k3_idx", "mp_band_vec_k3_strip_s1_idx", "mp_band_vec_k3_strip_s2_idx"}}}};
            *variant = names[a.idx ? 1 : 0][vec ? 1 : 0][k == 0 ? 0 : k - 1][sv];
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
