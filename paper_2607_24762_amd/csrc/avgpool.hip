// avgpool.hip -- adaptive_avg_pool2d for gfx950 (PyTorch semantics: output
// cell (i, j) averages input rows [floor(i*H/OH), ceil((i+1)*H/OH)) and
// columns [floor(j*W/OW), ceil((j+1)*W/OW))), the operator behind the
// paper's ResNet-50 adaptive_avgpool2d result (Section IV-C).
//
//   ap_flat   1x1 output, planes of S = H*W elements.  A workgroup owns P
//             consecutive planes = one contiguous span of P*S <= 4096
//             elements, which it stages in LDS with coalesced (16-byte when
//             aligned) loads, all issued before the first LDS store; then
//             TPS = 256/P threads sum each plane out of LDS and one of them
//             writes the mean.
//   ap_plane  1x1 output for large planes: one workgroup per plane reads it
//             with coalesced loads and reduces in registers.
//   ap_staged any output size, planes of at most 4096 elements: P planes
//             staged in LDS as in ap_flat, then one thread per output cell
//             sums its window from LDS.
//   ap_window any output size, larger planes: one thread per output cell.
//   ap_nhwc_cell  channels last, windows of at most 4 x 4: a thread per
//             output cell and 16-byte channel vector.
//   ap_nhwc   channels last, any output size: a workgroup owns one output
//             cell of one sample and 32 vectors of 16 bytes of channels;
//             its 16 thread groups sum interleaved window pixels, so every
//             load is a coalesced 512-byte channel run, and the 16 partials
//             are added in group order through LDS.
#include <algorithm>
#include <type_traits>

#include "kf_device.hpp"
#include "kf_internal.h"

namespace kf {
namespace {

constexpr int kNT = 256;
constexpr int kSpanMax = 4096;  // fp32 staging per workgroup: 16 KiB of LDS
constexpr int64_t kStagedBlocks = 2048;  // ap_staged: target workgroups (1024-4096 measured alike)

// Loads issued per thread to cover a span of kSpanMax elements.
template <int VEC>
constexpr int slots() {
    return (kSpanMax + kNT * VEC - 1) / (kNT * VEC);
}

// Stage elements [base, base + span) of x in LDS as fp32 (span <= kSpanMax).
// Every load is issued before the first LDS store, so a thread has all its
// requests in flight at once (non-temporal: the span is read once); only
// the last workgroup can have a remainder that is not whole vectors (VECTOR
// needs x + base 16-byte aligned).  A lane
// writes its four fp32 values with one 16-byte LDS store: as 4-byte stores,
// lanes 16 apart would hit the same bank.  Ends with a barrier.
template <class T, bool VECTOR>
__device__ __forceinline__ void stage_span(const void* __restrict__ x, int64_t base, int32_t span, float4* tile4) {
    constexpr int VEC = VECTOR ? T::vec : 1;
    constexpr int NV = slots<VEC>();
    float* tile = reinterpret_cast<float*>(tile4);
    const int32_t whole = span - span % VEC;
    float v[NV][VEC];
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        const int32_t e = (k * kNT + (int)threadIdx.x) * VEC;
        if (e < whole) {
            if constexpr (VECTOR) load_vec<T, true>(x, base + e, v[k]);
            else v[k][0] = load1<T>(x, base + e);
        }
    }
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        const int32_t e = (k * kNT + (int)threadIdx.x) * VEC;
        if (e < whole) {
            if constexpr (VEC % 4 == 0) {
#pragma unroll
                for (int i = 0; i < VEC; i += 4)
                    tile4[(e + i) / 4] = make_float4(v[k][i], v[k][i + 1], v[k][i + 2], v[k][i + 3]);
            } else {
                tile[e] = v[k][0];
            }
        }
    }
    for (int32_t e = whole + threadIdx.x; e < span; e += kNT) tile[e] = load1<T>(x, base + e);
    __syncthreads();
}

template <class T, int TPS, bool VECTOR>
__global__ __launch_bounds__(kNT) void ap_flat(const void* __restrict__ x, void* __restrict__ y, int64_t planes,
                                               int32_t S) {
    constexpr int P = kNT / TPS;  // planes per workgroup
    extern __shared__ float4 tile4[];  // P * S floats, 16-byte aligned
    float* tile = reinterpret_cast<float*>(tile4);
    const int64_t p0 = (int64_t)blockIdx.x * P;
    const int64_t np = (planes - p0) < P ? (planes - p0) : P;
    stage_span<T, VECTOR>(x, p0 * S, (int32_t)(np * S), tile4);

    // TPS threads sum each plane at stride TPS, four accumulators each.
    const int q = threadIdx.x / TPS;
    const int part = threadIdx.x % TPS;
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    if (q < np) {
        const float* row = tile + q * S;
        int32_t j = part;
        for (; j + 3 * TPS < S; j += 4 * TPS) {
            acc[0] += row[j];
            acc[1] += row[j + TPS];
            acc[2] += row[j + 2 * TPS];
            acc[3] += row[j + 3 * TPS];
        }
        for (int r = 0; j < S; j += TPS, ++r) acc[r] += row[j];
    }
    float sum = (acc[0] + acc[1]) + (acc[2] + acc[3]);
    sum = group_reduce<TPS>(sum, OpSum{});
    if (part == 0 && q < np) store1<T>(y, p0 + q, sum / (float)S);
}

template <class T, bool VECTOR>
__global__ __launch_bounds__(kNT) void ap_plane(const void* __restrict__ x, void* __restrict__ y, int64_t S) {
    constexpr int VEC = VECTOR ? T::vec : 1;
    constexpr int DEPTH = 4;  // loads in flight per thread per iteration
    __shared__ float red[kNT / kWave];
    const int64_t base = (int64_t)blockIdx.x * S;
    float acc[DEPTH] = {0.f, 0.f, 0.f, 0.f};
    for (int64_t e0 = (int64_t)threadIdx.x * VEC; e0 < S; e0 += (int64_t)DEPTH * kNT * VEC) {
        float v[DEPTH][VEC];
#pragma unroll
        for (int d = 0; d < DEPTH; ++d) {
            const int64_t e = e0 + (int64_t)d * kNT * VEC;
            if (e < S) {
                if constexpr (VECTOR) load_vec<T>(x, base + e, v[d]);
                else v[d][0] = load1<T>(x, base + e);
            } else {
#pragma unroll
                for (int i = 0; i < VEC; ++i) v[d][i] = 0.f;
            }
        }
#pragma unroll
        for (int d = 0; d < DEPTH; ++d)
#pragma unroll
            for (int i = 0; i < VEC; ++i) acc[d] += v[d][i];
    }
    float sum = (acc[0] + acc[1]) + (acc[2] + acc[3]);
    sum = group_reduce<kWave>(sum, OpSum{});
    if ((threadIdx.x & (kWave - 1)) == 0) red[threadIdx.x / kWave] = sum;
    __syncthreads();
    if (threadIdx.x == 0) {
        float t = red[0];
#pragma unroll
        for (int i = 1; i < kNT / kWave; ++i) t += red[i];
        store1<T>(y, blockIdx.x, t / (float)S);
    }
}

// Any output size, planes of S = H * W <= kSpanMax elements: a workgroup
// stages P consecutive planes (one contiguous span) in LDS as ap_flat does,
// then its threads take the P * OH * OW output cells in order (consecutive
// threads, consecutive cells, coalesced stores) and sum each window from LDS
// row by row.  Window bounds are PyTorch's adaptive ones, computed once per
// workgroup into LDS tables (row i: h0 | h1 << 16, column j: w0 | w1 << 16;
// every bound is at most 4096); a thread steps its (plane, row, column) by
// the workgroup size with carries instead of dividing per cell.  KMAX > 0:
// no window is more than KMAX rows or columns, and the window is read as a
// fixed KMAX x KMAX block (reads outside the window clamped and added as 0,
// in the same row-major order), so its LDS reads issue together instead of
// one loop trip and one wait each.
template <class T, bool VECTOR, int KMAX>
__global__ __launch_bounds__(kNT) void ap_staged(const void* __restrict__ x, void* __restrict__ y, int64_t planes,
                                                 int32_t P, int32_t H, int32_t W, int32_t OH, int32_t OW) {
    extern __shared__ float4 tile4[];  // P * H * W floats, then OH + OW bounds
    const float* tile = reinterpret_cast<const float*>(tile4);
    const int32_t S = H * W, cells = OH * OW;
    uint32_t* rows = reinterpret_cast<uint32_t*>(reinterpret_cast<float*>(tile4) + P * S);
    uint32_t* cols = rows + OH;
    for (int32_t t = threadIdx.x; t < OH + OW; t += kNT) {
        const int32_t k = t < OH ? t : t - OH, n = t < OH ? H : W, m = t < OH ? OH : OW;
        rows[t] = (uint32_t)((k * n) / m) | ((uint32_t)(((k + 1) * n + m - 1) / m) << 16);
    }
    const int64_t p0 = (int64_t)blockIdx.x * P;
    const int32_t np = (int32_t)((planes - p0) < P ? (planes - p0) : P);
    stage_span<T, VECTOR>(x, p0 * S, np * S, tile4);  // its barrier also publishes the tables
    // This thread's first cell, and the step kNT = dq * cells + di * OW + dj.
    int32_t q = (int32_t)threadIdx.x / cells;
    int32_t i = ((int32_t)threadIdx.x - q * cells) / OW;
    int32_t j = (int32_t)threadIdx.x - q * cells - i * OW;
    const int32_t dq = kNT / cells, di = (kNT - dq * cells) / OW, dj = kNT - dq * cells - di * OW;
    for (int32_t o = threadIdx.x; o < np * cells; o += kNT) {
        const uint32_t rb = rows[i], cb = cols[j];
        const int32_t h0 = (int32_t)(rb & 0xffff), h1 = (int32_t)(rb >> 16);
        const int32_t w0 = (int32_t)(cb & 0xffff), w1 = (int32_t)(cb >> 16);
        const float* plane = tile + q * S;
        float sum = 0.f;
        if constexpr (KMAX > 0) {
            float v[KMAX][KMAX];
#pragma unroll
            for (int a = 0; a < KMAX; ++a)
#pragma unroll
                for (int b = 0; b < KMAX; ++b)
                    v[a][b] = plane[min(h0 + a, H - 1) * W + min(w0 + b, W - 1)];
#pragma unroll
            for (int a = 0; a < KMAX; ++a)
#pragma unroll
                for (int b = 0; b < KMAX; ++b) sum += (h0 + a < h1 && w0 + b < w1) ? v[a][b] : 0.f;
        } else {
            for (int32_t rr = h0; rr < h1; ++rr)
                for (int32_t c = w0; c < w1; ++c) sum += plane[rr * W + c];
        }
        store1<T>(y, p0 * cells + o, sum / (float)((h1 - h0) * (w1 - w0)));
        j += dj;
        const int32_t cj = j >= OW;
        j -= cj * OW;
        i += di + cj;
        const int32_t ci = i >= OH;
        i -= ci * OH;
        q += dq + ci;
    }
}

template <class T>
__global__ __launch_bounds__(kNT) void ap_window(const void* __restrict__ x, void* __restrict__ y, int64_t planes,
                                                 int64_t H, int64_t W, int64_t OH, int64_t OW) {
    const int64_t idx = (int64_t)blockIdx.x * kNT + threadIdx.x;
    if (idx >= planes * OH * OW) return;
    const int64_t j = idx % OW;
    const int64_t i = (idx / OW) % OH;
    const int64_t p = idx / (OW * OH);
    const int64_t h0 = (i * H) / OH, h1 = ((i + 1) * H + OH - 1) / OH;
    const int64_t w0 = (j * W) / OW, w1 = ((j + 1) * W + OW - 1) / OW;
    const int64_t base = p * H * W;
    float sum = 0.f;
    for (int64_t r = h0; r < h1; ++r)
        for (int64_t c = w0; c < w1; ++c) sum += load1<T>(x, base + r * W + c);
    store1<T>(y, idx, sum / (float)((h1 - h0) * (w1 - w0)));
}

// ap_nhwc: a workgroup owns kCB consecutive 16-byte channel vectors of one
// output cell of one sample; its kPG thread groups take the window's pixels
// g, g + kPG, ... (kPD of them per thread per batch, every load of a batch
// issued before the first add), and the groups' sums meet in LDS in group
// order.  Consecutive threads read consecutive channel vectors, so each
// pixel is a 512-byte run.  On the channels-last ResNet-50 head ([32, 2048,
// 7, 7] fp32 -> 1x1, graph replays, one box): 5.82 us for the earlier 64 x 4
// shape with 16 loads per thread in flight (three of them re-reading pixel 0
// past the window's 13), 4.76 us for 64 x 4 with the loads here, 4.40 us
// for 32 x 16 (16 x 16: 4.66, 16 x 32: 4.69, 32 x 32: 4.63, 128 x 8: 5.03),
// against 3.78 us for a plain read of the 12.25 MiB.  Loads are non-temporal
// where the windows tile the input (every pixel read once: 4.40 against 4.55
// us with ordinary loads), ordinary where adaptive windows overlap.
constexpr int kCB = 32;               // channel vectors per ap_nhwc workgroup
constexpr int kPG = 16;               // pixel groups per workgroup
constexpr int kPD = 4;                // window pixels per thread per batch
constexpr int kNhwcNT = kCB * kPG;    // 512 threads

template <class T, int VEC, bool NT>
__global__ __launch_bounds__(kNhwcNT) void ap_nhwc(const void* __restrict__ x, void* __restrict__ y, int32_t H,
                                                   int32_t W, int32_t C, int32_t OH, int32_t OW) {
    __shared__ float part[kPG - 1][kCB][VEC];
    const int lc = threadIdx.x % kCB, g = threadIdx.x / kCB;
    const int cv = blockIdx.x * kCB + lc;
    const bool active = cv < C / VEC;
    const int i = blockIdx.y / OW, j = blockIdx.y - (blockIdx.y / OW) * OW;
    const int64_t n = blockIdx.z;
    // Window bounds; a 1 x 1 output's window is the whole plane, with none
    // of the 64-bit divisions (hundreds of instructions ahead of the loads).
    int h0 = 0, h1 = H, w0 = 0, w1 = W;
    if (OH != 1 || OW != 1) {
        h0 = (int)(((int64_t)i * H) / OH), h1 = (int)((((int64_t)i + 1) * H + OH - 1) / OH);
        w0 = (int)(((int64_t)j * W) / OW), w1 = (int)((((int64_t)j + 1) * W + OW - 1) / OW);
    }
    const int ww = w1 - w0, count = (h1 - h0) * ww;
    const int64_t base = n * H * W * (int64_t)C + (int64_t)cv * VEC;
    // Pixel q of the window, row-major; a window spanning whole rows (every
    // 1 x 1 or one-column output) is one run of pixels, with no division.
    const bool rows = ww == W;
    auto at = [&](int q) {
        if (rows) return base + ((int64_t)h0 * W + q) * C;
        const int r = h0 + q / ww, c = w0 + (q - (q / ww) * ww);
        return base + ((int64_t)r * W + c) * C;
    };
    float acc[VEC];
#pragma unroll
    for (int k = 0; k < VEC; ++k) acc[k] = 0.f;
    if (active) {
        // A slot past the window re-reads the window's first pixel and is
        // not added.
        for (int q0 = g; q0 < count; q0 += kPD * kPG) {
            float v[kPD][VEC];
#pragma unroll
            for (int d = 0; d < kPD; ++d) {
                const int q = q0 + d * kPG;
                const int64_t e = at(q < count ? q : 0);
                if constexpr (VEC > 1) load_vec<T, NT>(x, e, v[d]);
                else v[d][0] = load1<T>(x, e);
            }
#pragma unroll
            for (int d = 0; d < kPD; ++d)
                if (q0 + d * kPG < count) {
#pragma unroll
                    for (int k = 0; k < VEC; ++k) acc[k] += v[d][k];
                }
        }
    }
    if (g > 0) {
#pragma unroll
        for (int k = 0; k < VEC; ++k) part[g - 1][lc][k] = acc[k];
    }
    __syncthreads();
    if (g == 0 && active) {
        const float cnt = (float)count;
#pragma unroll
        for (int k = 0; k < VEC; ++k) {
            float s = acc[k];
#pragma unroll
            for (int gg = 0; gg < kPG - 1; ++gg) s += part[gg][lc][k];
            acc[k] = s / cnt;
        }
        const int64_t o = ((n * OH + i) * OW + j) * (int64_t)C + (int64_t)cv * VEC;
        if constexpr (VEC > 1) store_vec<T, false>(y, o, acc);
        else store1<T>(y, o, acc[0]);
    }
}

// Channels last, windows of at most K x K pixels (ap_nhwc_cell): one thread
// per (sample, output cell, 16-byte channel vector), consecutive threads on
// consecutive channel vectors, so every window pixel is read as a coalesced
// run of channels.  The K x K block is read from clamped addresses (a pixel
// past the window repeats the window's last row or column), all loads
// issued before the adds, and the pixels inside the window are added in
// row-major order.  No LDS and no barrier: small windows leave too little
// work per output cell to split it over thread groups as ap_nhwc does.
// I32: the thread index, the products i * H and j * W and their bounds fit
// in 32 bits (checked on the host), so the index arithmetic divides in 32
// bits: seven 64-bit divisions by run-time values cost about a thousand
// VALU instructions per thread ahead of the loads.
template <class I>
__device__ __forceinline__ void cell_of(I idx, I CV, I OH, I OW, I H, I W, int* cv, int* i, int* j, int64_t* n,
                                        int* h0, int* h1, int* w0, int* w1) {
    const I cell = idx / CV, t = cell / OW;
    *cv = (int)(idx - cell * CV);
    *j = (int)(cell - t * OW);
    *n = (int64_t)(t / OH);
    *i = (int)(t - (t / OH) * OH);
    *h0 = (int)(((I)*i * H) / OH), *h1 = (int)((((I)*i + 1) * H + OH - 1) / OH);
    *w0 = (int)(((I)*j * W) / OW), *w1 = (int)((((I)*j + 1) * W + OW - 1) / OW);
}

template <class T, int VEC, int K, bool I32>
__global__ __launch_bounds__(kNT) void ap_nhwc_cell(const void* __restrict__ x, void* __restrict__ y, int64_t total,
                                                    int32_t CV, int32_t H, int32_t W, int32_t C, int32_t OH,
                                                    int32_t OW) {
    const int64_t idx = (int64_t)blockIdx.x * kNT + threadIdx.x;
    if (idx >= total) return;
    int cv, i, j, h0, h1, w0, w1;
    int64_t n;
    if constexpr (I32)
        cell_of<uint32_t>((uint32_t)idx, CV, OH, OW, H, W, &cv, &i, &j, &n, &h0, &h1, &w0, &w1);
    else
        cell_of<int64_t>(idx, CV, OH, OW, H, W, &cv, &i, &j, &n, &h0, &h1, &w0, &w1);
    const int hh = h1 - h0, ww = w1 - w0;
    const int64_t base = n * H * W * (int64_t)C + (int64_t)cv * VEC;
    float v[K][K][VEC];
#pragma unroll
    for (int a = 0; a < K; ++a)
#pragma unroll
        for (int b = 0; b < K; ++b) {
            const int r = h0 + (a < hh ? a : hh - 1), c = w0 + (b < ww ? b : ww - 1);
            const int64_t e = base + ((int64_t)r * W + c) * C;
            if constexpr (VEC > 1) load_vec<T>(x, e, v[a][b]);
            else v[a][b][0] = load1<T>(x, e);
        }
    float acc[VEC];
#pragma unroll
    for (int k = 0; k < VEC; ++k) acc[k] = 0.f;
#pragma unroll
    for (int a = 0; a < K; ++a)
#pragma unroll
        for (int b = 0; b < K; ++b)
            if (a < hh && b < ww) {
#pragma unroll
                for (int k = 0; k < VEC; ++k) acc[k] += v[a][b][k];
            }
    const float cnt = (float)(hh * ww);
#pragma unroll
    for (int k = 0; k < VEC; ++k) acc[k] = acc[k] / cnt;
    const int64_t o = ((n * OH + i) * OW + j) * (int64_t)C + (int64_t)cv * VEC;
    if constexpr (VEC > 1) store_vec<T, false>(y, o, acc);
    else store1<T>(y, o, acc[0]);
}

// Largest window extent of an adaptive pooling of n positions into m.
int64_t window_extent(int64_t n, int64_t m) {
    int64_t e = 0;
    for (int64_t k = 0; k < m; ++k) {
        const int64_t d = ((k + 1) * n + m - 1) / m - (k * n) / m;
        e = d > e ? d : e;
    }
    return e;
}

template <class T, int TPS>
void launch_flat(const AvgPoolArgs& a, hipStream_t s, const char** variant, const char* name) {
    constexpr int P = kNT / TPS;
    const int64_t S = a.h * a.w;
    const int64_t blocks = (a.planes + P - 1) / P;
    const size_t lds = (size_t)P * S * sizeof(float);
    // Vector loads need every workgroup span to start 16-byte aligned.
    const bool vec = ((P * S * T::bytes) % 16 == 0) && ((uintptr_t)a.x % 16 == 0);
    if (vec)
        hipLaunchKernelGGL((ap_flat<T, TPS, true>), dim3((unsigned)blocks), dim3(kNT), lds, s, a.x, a.y, a.planes,
                           (int32_t)S);
    else
        hipLaunchKernelGGL((ap_flat<T, TPS, false>), dim3((unsigned)blocks), dim3(kNT), lds, s, a.x, a.y,
                           a.planes, (int32_t)S);
    *variant = name;
}

template <class T>
kf_status run(const AvgPoolArgs& a, hipStream_t s, const char** variant) {
    const int64_t S = a.h * a.w;
    if (a.nhwc) {
        const bool vec = a.c % T::vec == 0 && (uintptr_t)a.x % 16 == 0 && (uintptr_t)a.y % 16 == 0;
        const int64_t cvs = vec ? a.c / T::vec : a.c;
        const int64_t gx = (cvs + kCB - 1) / kCB, gy = a.oh * a.ow;
        if (gx > INT32_MAX || gy > INT32_MAX || a.n > 65535 || a.h * a.w * a.c > INT64_MAX / 2 ||
            a.h > INT32_MAX || a.w > INT32_MAX || a.c > INT32_MAX) {
            set_error("adaptive_avgpool2d: channels-last problem exceeds the grid limits");
            return KF_ERR_UNSUPPORTED_LAYOUT;
        }
        // Windows of at most 4 x 4 pixels: a thread per output cell and
        // channel vector ([32, 512, 14, 14] -> 7 x 7: 16.0 us with ap_nhwc's
        // split windows, which suit large windows such as the 7 x 7 -> 1 x 1
        // head).
        const int64_t ext = (a.oh <= 4096 && a.ow <= 4096)
                                ? std::max(window_extent(a.h, a.oh), window_extent(a.w, a.ow)) : 0;
        const int kc = ext == 0 ? 0 : ext <= 2 ? 2 : ext <= 3 ? 3 : ext <= 4 ? 4 : 0;
        const int64_t total = a.n * a.oh * a.ow * cvs;
        if (kc > 0 && (total + kNT - 1) / kNT <= INT32_MAX) {
            const unsigned blocks = (unsigned)((total + kNT - 1) / kNT);
            auto go = [&](auto kernel) {
                hipLaunchKernelGGL(kernel, dim3(blocks), dim3(kNT), 0, s, a.x, a.y, total, (int32_t)cvs,
                                   (int32_t)a.h, (int32_t)a.w, (int32_t)a.c, (int32_t)a.oh, (int32_t)a.ow);
            };
            const bool i32 = total <= INT32_MAX && (a.oh + 1) * (a.h + 1) <= INT32_MAX && (a.ow + 1) * (a.w + 1) <= INT32_MAX;
            auto pick = [&](auto vec_tag) {
                constexpr int V = decltype(vec_tag)::value;
                if (i32) {
                    if (kc == 2) go(ap_nhwc_cell<T, V, 2, true>);
                    else if (kc == 3) go(ap_nhwc_cell<T, V, 3, true>);
                    else go(ap_nhwc_cell<T, V, 4, true>);
                } else {
                    if (kc == 2) go(ap_nhwc_cell<T, V, 2, false>);
                    else if (kc == 3) go(ap_nhwc_cell<T, V, 3, false>);
                    else go(ap_nhwc_cell<T, V, 4, false>);
                }
            };
            if (vec) pick(std::integral_constant<int, T::vec>{});
            else pick(std::integral_constant<int, 1>{});
            static const char* names[2][5] = {
                {"", "", "ap_nhwc_cell_scalar_k2", "ap_nhwc_cell_scalar_k3", "ap_nhwc_cell_scalar_k4"},
                {"", "", "ap_nhwc_cell_vec_k2", "ap_nhwc_cell_vec_k3", "ap_nhwc_cell_vec_k4"}};
            *variant = names[vec ? 1 : 0][kc];
            const hipError_t err = hipGetLastError();
            if (err != hipSuccess) {
                set_error("adaptive_avgpool2d launch failed: %s", hipGetErrorString(err));
                return KF_ERR_HIP;
            }
            return KF_OK;
        }
        const dim3 grid((unsigned)gx, (unsigned)gy, (unsigned)a.n), block(kNhwcNT);
        const bool tiled = a.h % a.oh == 0 && a.w % a.ow == 0;  // windows tile x: every pixel read once
        auto go = [&](auto kernel) {
            hipLaunchKernelGGL(kernel, grid, block, 0, s, a.x, a.y, (int32_t)a.h, (int32_t)a.w, (int32_t)a.c,
                               (int32_t)a.oh, (int32_t)a.ow);
        };
        if (vec) tiled ? go(ap_nhwc<T, T::vec, true>) : go(ap_nhwc<T, T::vec, false>);
        else go(ap_nhwc<T, 1, false>);
        *variant = vec ? "ap_nhwc_vec" : "ap_nhwc_scalar";
    } else if (a.oh == 1 && a.ow == 1) {
        // Planes per workgroup: the largest power of two (<= 256) whose span
        // fits the staging tile; a plane too big for it gets a workgroup.
        int64_t P = 256;
        while (P > 1 && P * S > kSpanMax) P /= 2;
        if (P * S > kSpanMax) P = 0;
        if (P > 0 && (a.planes + P - 1) / P > INT32_MAX) P = 0;
        switch (P) {
            case 256: launch_flat<T, 1>(a, s, variant, "ap_flat_tps1"); break;
            case 128: launch_flat<T, 2>(a, s, variant, "ap_flat_tps2"); break;
            case 64: launch_flat<T, 4>(a, s, variant, "ap_flat_tps4"); break;
            case 32: launch_flat<T, 8>(a, s, variant, "ap_flat_tps8"); break;
            case 16: launch_flat<T, 16>(a, s, variant, "ap_flat_tps16"); break;
            case 8: launch_flat<T, 32>(a, s, variant, "ap_flat_tps32"); break;
            case 4: launch_flat<T, 64>(a, s, variant, "ap_flat_tps64"); break;
            default: {
                if (a.planes > INT32_MAX) {
                    set_error("adaptive_avgpool2d: %lld planes exceed the grid limit", (long long)a.planes);
                    return KF_ERR_UNSUPPORTED_LAYOUT;
                }
                const bool vec = (S % T::vec == 0) && ((uintptr_t)a.x % 16 == 0);
                if (vec)
                    hipLaunchKernelGGL((ap_plane<T, true>), dim3((unsigned)a.planes), dim3(kNT), 0, s, a.x, a.y, S);
                else
                    hipLaunchKernelGGL((ap_plane<T, false>), dim3((unsigned)a.planes), dim3(kNT), 0, s, a.x, a.y,
                                       S);
                *variant = "ap_plane";
            }
        }
    } else if (S <= kSpanMax && a.oh + a.ow <= 4096 &&
               (kSpanMax / S) * a.oh * a.ow <= INT32_MAX && (a.planes + kSpanMax / S - 1) / (kSpanMax / S) <= INT32_MAX) {
        // Planes per workgroup: as many as fit the staging tile, but no more
        // than leave kStagedBlocks workgroups (enough to keep every CU busy
        // with several), rounded down so the span stays whole 16-byte vectors
        // when it can.
        int64_t P = kSpanMax / S;
        const int64_t spread = a.planes / kStagedBlocks;
        P = spread < 1 ? 1 : (spread < P ? spread : P);
        const int64_t vec_elems = T::vec;
        while (P > 1 && (P * S) % vec_elems != 0) --P;
        const int64_t blocks = (a.planes + P - 1) / P;
        const bool vec = ((P * S) % vec_elems == 0) && ((uintptr_t)a.x % 16 == 0);
        const size_t lds = (size_t)(P * S) * sizeof(float) + (size_t)(a.oh + a.ow) * sizeof(uint32_t);
        // Largest window extent along either axis.
        const int64_t ext = std::max(window_extent(a.h, a.oh), window_extent(a.w, a.ow));
        const int kmax = ext <= 2 ? 2 : ext <= 3 ? 3 : ext <= 4 ? 4 : 0;
        auto go = [&](auto kernel) {
            hipLaunchKernelGGL(kernel, dim3((unsigned)blocks), dim3(kNT), lds, s, a.x, a.y, a.planes, (int32_t)P,
                               (int32_t)a.h, (int32_t)a.w, (int32_t)a.oh, (int32_t)a.ow);
        };
        auto pick = [&](auto vec_tag) {
            constexpr bool V = decltype(vec_tag)::value;
            if (kmax == 2) go(ap_staged<T, V, 2>);
            else if (kmax == 3) go(ap_staged<T, V, 3>);
            else if (kmax == 4) go(ap_staged<T, V, 4>);
            else go(ap_staged<T, V, 0>);
        };
        if (vec) pick(std::true_type{});
        else pick(std::false_type{});
        static const char* names[2][5] = {
            {"ap_staged_scalar", "", "ap_staged_scalar_k2", "ap_staged_scalar_k3", "ap_staged_scalar_k4"},
            {"ap_staged_vec", "", "ap_staged_vec_k2", "ap_staged_vec_k3", "ap_staged_vec_k4"}};
        *variant = names[vec ? 1 : 0][kmax];
    } else {
        const int64_t blocks = (a.planes * a.oh * a.ow + kNT - 1) / kNT;
        if (blocks > INT32_MAX) {
            set_error("adaptive_avgpool2d: problem exceeds the grid limit");
            return KF_ERR_UNSUPPORTED_LAYOUT;
        }
        hipLaunchKernelGGL((ap_window<T>), dim3((unsigned)blocks), dim3(kNT), 0, s, a.x, a.y, a.planes, a.h, a.w,
                           a.oh, a.ow);
        *variant = "ap_window";
    }
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) {
        set_error("adaptive_avgpool2d launch failed: %s", hipGetErrorString(err));
        return KF_ERR_HIP;
    }
    return KF_OK;
}

}  // namespace

kf_status avgpool_launch(const AvgPoolArgs& a, hipStream_t s, const char** variant) {
    switch (a.t) {
        case KF_FLOAT32:
            return run<F32>(a, s, variant);
        case KF_BFLOAT16:
            return run<BF16>(a, s, variant);
        case KF_FLOAT16:
            return run<F16>(a, s, variant);
    }
    set_error("adaptive_avgpool2d: unsupported dtype");
    return KF_ERR_BAD_DTYPE;
}

}  // namespace kf
