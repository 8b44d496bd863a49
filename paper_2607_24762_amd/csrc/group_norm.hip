// group_norm.hip -- GroupNorm for gfx950 (PyTorch `group_norm(x, G, w, b,
// eps)` semantics: biased variance, eps inside the square root, per-channel
// affine), the operator behind the paper's SD3.5 Medium group_norm result
// (Section IV-C).
//
// Layout: x is dense [n, c, spatial] (NCHW) or dense [n, spatial, c]
// (channels last).  A group's (c/G)*spatial elements are numbered o = 0, 1,
// ...: NCHW in memory order (the group is one contiguous span), channels
// last pixel-major (element o is channel g*cpg + o % cpg of pixel o / cpg),
// so VEC consecutive elements are VEC adjacent channels of one pixel: 16
// contiguous bytes either way.  Each group is cut into `parts` chunks of
// CH = 256 threads * NV * VEC elements and one workgroup owns one chunk.
//
//   gn_pipe   (one launch, one HBM read + one write; dense NCHW 16-bit
//             tensors whose spatial size is a multiple of 2048)  Four data
//             waves hold the chunk as raw 16-bit pairs and fold its moments
//             with v_dot2; a fifth wave, which has no loads of the tensor
//             outstanding, does the whole exchange (publish, poll, merge,
//             affine, departure), so its polls never wait behind chunk
//             loads.  Described at the kernel below.
//   gn_fused  (one launch, one HBM read + one write)  Each workgroup keeps its
//             chunk in registers, computes its (count, mean, M2) moments,
//             publishes them as one 64-bit word in its workspace slot, polls
//             the slots of its group until all `parts` are published, merges
//             them in part order (so the result does not depend on arrival
//             order), and normalises straight from registers.  Needs every
//             workgroup of the grid resident at once.
//   gn_split  (two launches; dense NCHW 16-bit tensors gn_pipe cannot take)
//             gn_pipe's chunks and arithmetic without any wait: the first
//             launch publishes each chunk's moments and the group's last
//             arrival merges them; the second re-reads x and normalises.
//   gn_stats + gn_apply  (two launches)  gn_fused's chunking without the
//             wait: the first kernel publishes the partials, the second
//             merges them and re-reads x.  Used for the other grids that
//             cannot be co-resident.
//
// Moments: each thread computes its own mean and M2 by two passes over its
// registers, then partials are combined with the Chan et al. parallel
// update; both lanes of a butterfly pair order the operands by lane so they
// compute bit-identical results.
#include <math.h>

#include <atomic>
#include <cstdlib>
#include <cstring>
#include <type_traits>

#include "kf_device.hpp"
#include "kf_exchange.hpp"
#include "kf_internal.h"

namespace kf {
namespace {

constexpr int kNT = 256;          // threads per workgroup
constexpr int kFloatsPerThread = 64;

struct GNParams {
    const void* x;
    void* y;
    const void* w;
    const void* b;
    Exchange ex;           // one unit per (sample, group), ex.parts chunks each
    int64_t group_elems;   // (c/G) * spatial
    int64_t spatial;
    int64_t channels;      // c
    int32_t cpg;           // channels per group
    int32_t groups;        // G
    int32_t xcd_map;       // 1: place all parts of a group on one XCD (block_chunk)
    float eps;
};

// The (group, part) chunk that workgroup b handles.  Workgroups are handed
// to the 8 XCDs in turn (b % 8); when the number of groups is a multiple of
// 8, every part of group ng runs on XCD ng % 8, so a group's exchange and
// the moment its last part lands stay within one XCD (measured ~1% faster
// on the SD3.5 VAE block than groups spread over all eight); otherwise the
// plain order b = group * parts + part.  Channels last keeps the plain
// order: there neighbouring groups share every cache line (a 128-byte line
// holds four groups of 16 bf16 channels), and with parts a multiple of 8
// the plain order puts part q of every group on XCD q % 8, so each line is
// fetched into one L2; the one-XCD-per-group order fetched every line into
// four L2s (4x the input from HBM, 24 us against 16 us).
__device__ __forceinline__ void block_chunk(const GNParams& p, int64_t b, int64_t* ng, int* part) {
    if (p.xcd_map) {
        const int64_t slot = b >> 3;
        *ng = (b & 7) + 8 * (slot / p.ex.parts);
        *part = (int)(slot - (slot / p.ex.parts) * p.ex.parts);
    } else {
        *ng = b / p.ex.parts;
        *part = (int)(b - *ng * p.ex.parts);
    }
}

// What an absent weight (element 0) or bias (element 1) reads, in each
// affine storage type.  The affine loads read these instead of branching on
// the pointers: inside a branch, the conversion of the loaded values made
// the compiler wait for every outstanding load (the chunk's too) before the
// branch could end, so each workgroup paid an extra load round trip before
// it could publish its moments.  Plain (not const) device globals, so the
// pointer chosen between them and a kernel argument stays in the global
// address space and the loads remain global loads.  Never written.
__device__ float kIdentityF32[2] = {1.f, 0.f};
__device__ uint16_t kIdentityBF16[2] = {0x3F80u, 0u};
__device__ uint16_t kIdentityF16[2] = {0x3C00u, 0u};
template <class A>
__device__ __forceinline__ const void* affine_identity();
template <>
__device__ __forceinline__ const void* affine_identity<F32>() {
    return kIdentityF32;
}
template <>
__device__ __forceinline__ const void* affine_identity<BF16>() {
    return kIdentityBF16;
}
template <>
__device__ __forceinline__ const void* affine_identity<F16>() {
    return kIdentityF16;
}

// Elements held by part p of a group.
__device__ __forceinline__ float part_count(const GNParams& p, int64_t chunk, int part) {
    const int64_t left = p.group_elems - (int64_t)part * chunk;
    return (float)(left < chunk ? left : chunk);
}

template <class T, bool VECTOR, bool NHWC>
struct Chunk {
    static constexpr int VEC = VECTOR ? T::vec : 1;
    static constexpr int NV = kFloatsPerThread / VEC;
    static constexpr int64_t CH = (int64_t)kNT * NV * VEC;
    float v[NV][VEC];

    // Offset inside the group of this thread's k-th slot.
    __device__ __forceinline__ static int64_t off(int part, int k) {
        return (int64_t)part * CH + ((int64_t)k * kNT + threadIdx.x) * VEC;
    }
    // Element index in x / y of offset o of group ng (= sample * G + g).  A
    // group holds fewer than 2^31 elements (checked on the host), so the
    // channels-last split of o is a 32-bit division.
    __device__ __forceinline__ static int64_t at(const GNParams& p, int64_t ng, int64_t o) {
        if constexpr (!NHWC) {
            return ng * p.group_elems + o;
        } else {
            const int64_t n = ng / p.groups;
            const int g = (int)(ng - n * p.groups);
            const uint32_t pix = (uint32_t)o / (uint32_t)p.cpg;
            const uint32_t ch = (uint32_t)o - pix * (uint32_t)p.cpg;
            return (n * p.spatial + pix) * p.channels + (int64_t)g * p.cpg + ch;
        }
    }
    // All slots load unconditionally so the loads issue back to back; a slot
    // past the group's end re-reads the group's first element and is never
    // used afterwards.  NT: non-temporal loads, for the read that is the
    // chunk's last.
    template <bool NT = false>
    __device__ __forceinline__ void load(const GNParams& p, int64_t ng, int part) {
#pragma unroll
        for (int k = 0; k < NV; ++k) {
            const int64_t o = off(part, k);
            const int64_t e = at(p, ng, o < p.group_elems ? o : 0);
            if constexpr (VECTOR) load_vec<T, NT>(p.x, e, v[k]);
            else v[k][0] = load1<T>(p.x, e);
        }
    }
    // Thread-local moments of the valid elements from sums shifted by K, the
    // mean of the thread's first slot (whose load lands first; a thread with
    // no valid slot holds copies of the group's first element there):
    // s1 = sum(x - K), s2 = sum((x - K)^2), mean = K + s1/n,
    // M2 = s2 - s1^2/n.  With K a sample mean of the same data the
    // subtraction keeps most of its digits (s1^2/n <= s2), and unlike a
    // two-pass form every element is folded in as soon as its load lands,
    // overlapping this work with the remaining loads.
    __device__ __forceinline__ Moments moments(const GNParams& p, int part) const {
        float K = v[0][0];
#pragma unroll
        for (int i = 1; i < VEC; ++i) K += v[0][i];
        K *= 1.f / (float)VEC;
        float s1 = 0.f, s2 = 0.f, cnt = 0.f;
#pragma unroll
        for (int k = 0; k < NV; ++k) {
            if (off(part, k) < p.group_elems) {
                cnt += (float)VEC;
#pragma unroll
                for (int i = 0; i < VEC; ++i) {
                    const float d = v[k][i] - K;
                    s1 += d;
                    s2 = fmaf(d, d, s2);
                }
            }
        }
        if (cnt == 0.f) return Moments{0.f, 0.f, 0.f};
        const float r = __builtin_amdgcn_rcpf(cnt);
        const float d1 = s1 * r;
        return Moments{cnt, K + d1, fmaxf(fmaf(-s1, d1, s2), 0.f)};
    }
    // Raw w[c] and b[c], loaded before the statistics are known (they do
    // not depend on them), so their latency hides behind the cross-workgroup
    // wait.  NCHW, and scalar channels last: the channel of each slot
    // (a 16-byte NCHW vector lies inside one channel).  Vector channels
    // last: element i of every slot of this thread is channel
    // g*cpg + (thread*VEC) % cpg + i (the host requires cpg | 256*VEC, so
    // the channels do not change from slot to slot): wv[i], bv[i] for
    // i < VEC.  A group holds fewer than 2^31 elements (checked on the
    // host), so the channel index is a 32-bit division.
    float wv[NV], bv[NV];
    static constexpr bool kFixedChannels = NHWC && VECTOR;
    template <class A>
    __device__ __forceinline__ void load_affine(const GNParams& p, int part, int g) {
        int64_t c[NV];
#pragma unroll
        for (int k = 0; k < NV; ++k) {
            const int64_t o = off(part, k);
            const uint32_t oc = o < p.group_elems ? (uint32_t)o : 0u;
            if constexpr (kFixedChannels)
                c[k] = (int64_t)g * p.cpg + (int64_t)((threadIdx.x * VEC) % (uint32_t)p.cpg) + (k < VEC ? k : 0);
            else if constexpr (NHWC)
                c[k] = (int64_t)g * p.cpg + (int64_t)(oc % (uint32_t)p.cpg);
            else
                c[k] = (int64_t)g * p.cpg + (int64_t)(oc / (uint32_t)p.spatial);
        }
        // No branch: nothing here waits, so the loads stay in flight until
        // normalise_store uses them.
        const bool hw = p.w != nullptr, hb = p.b != nullptr;
        const void* ws = hw ? p.w : affine_identity<A>();
        const void* bs = hb ? p.b : affine_identity<A>();
#pragma unroll
        for (int k = 0; k < NV; ++k) {
            wv[k] = load1<A>(ws, hw ? c[k] : 0);
            bv[k] = load1<A>(bs, hb ? c[k] : 1);
        }
    }
    // y = (x - mean) * (rstd * w[c]) + b[c] with rstd = 1 / sqrt(M2/n + eps),
    // non-temporal stores.  16-bit outputs evaluate it in fp32.  fp32
    // outputs evaluate it in double and round once: x - mean is exact there
    // and rstd * w[c] carries no fp32 rounding, so the output's error is one
    // fp32 rounding plus what the fp32 statistics carry (in fp32 the three
    // extra roundings reached 1e-6 at |y| ~ 5).
    static constexpr bool kF64Apply = std::is_same_v<T, F32>;
    using Acc = std::conditional_t<kF64Apply, double, float>;
    __device__ __forceinline__ void normalise_store(const GNParams& p, int64_t ng, int part, float mean,
                                                    float m2) {
        Acc rstd;
        if constexpr (kF64Apply) rstd = 1.0 / sqrt((double)m2 / (double)p.group_elems + (double)p.eps);
        else rstd = 1.f / sqrtf(m2 / (float)p.group_elems + p.eps);
        const Acc mu = (Acc)mean;
        Acc ai[VEC];
        if constexpr (kFixedChannels) {
#pragma unroll
            for (int i = 0; i < VEC; ++i) ai[i] = rstd * (Acc)wv[i];
        }
#pragma unroll
        for (int k = 0; k < NV; ++k) {
            const int64_t o = off(part, k);
            if (o < p.group_elems) {
                float out[VEC];
                if constexpr (kFixedChannels) {
#pragma unroll
                    for (int i = 0; i < VEC; ++i) out[i] = (float)fma((Acc)v[k][i] - mu, ai[i], (Acc)bv[i]);
                } else {
                    const Acc a = rstd * (Acc)wv[k];
#pragma unroll
                    for (int i = 0; i < VEC; ++i) out[i] = (float)fma((Acc)v[k][i] - mu, a, (Acc)bv[k]);
                }
                // Non-temporal stores for NCHW (each workgroup writes whole
                // lines).  Channels last, a group's 16-byte runs share their
                // lines with neighbouring groups written by other workgroups:
                // ordinary stores let L2 merge those before writing back
                // (non-temporal ones measured twice the HBM write traffic).
                if constexpr (VECTOR) store_vec<T, !NHWC>(p.y, at(p, ng, o), out);
                else store1<T>(p.y, at(p, ng, o), out[0]);
            }
        }
    }
};

// A published partial is one 64-bit word: mean bits low, M2 bits high with
// the sign bit forced on.  M2 is never negative, so the flag is free, and a
// published word is never 0, the value of an empty slot.  Writing the data
// and its ready flag in one single-copy-atomic store means a reader that sees
// the word sees the data: no fences, no cache write-back or invalidation.
__device__ __forceinline__ uint64_t encode(Moments m) {
    return (uint64_t)__float_as_uint(m.mean) | ((uint64_t)(__float_as_uint(m.m2) | 0x80000000u) << 32);
}
__device__ __forceinline__ Moments decode(uint64_t w, float n) {
    return Moments{n, __uint_as_float((uint32_t)w), __uint_as_float((uint32_t)(w >> 32) & 0x7fffffffu)};
}

// Gather and merge the partials of one group; called by a whole wave,
// result uniform across it.  Lane l takes parts l, l+64, ... in order and the
// butterfly keeps lane order, so the combine order depends on part index
// alone (bitwise-reproducible results).  With `wait`, each lane polls its
// slots until they are published or the exchange's wait bound has passed;
// *ok reports (uniformly) whether every slot arrived.
__device__ __forceinline__ Moments gather_parts(const GNParams& p, int64_t ng, int64_t chunk, bool wait,
                                                bool* ok) {
    Moments acc{0.f, 0.f, 0.f};
    const int lane = threadIdx.x & (kWave - 1);
    const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
    bool all = true;
    for (int q = lane; q < p.ex.parts; q += kWave) {
        const uint64_t w = ex_poll(p.ex, ng, q, t0, wait);
        all = all && (w != 0);
        acc = chan(acc, decode(w, part_count(p, chunk, q)));
    }
    *ok = __all(all);
    return moments_wave(acc);
}

// The statistics of group ng for chunk c (part `part` of the group, whose
// own moments `own` the caller has already published when the group has
// several parts), then the normalised chunk, then the group's slots
// released.  Called by the whole workgroup; `stats` and `gathered` are LDS.
template <class C>
__device__ __forceinline__ void settle(const GNParams& p, C& c, int64_t ng, int part, Moments own, Moments* lds,
                                       float* stats, int* gathered) {
    if (threadIdx.x < kWave) {
        bool ok = true;
        Moments m = own;
        if (p.ex.parts > 1) m = gather_parts(p, ng, C::CH, true, &ok);
        if (threadIdx.x == 0) {
            *gathered = ok;
            stats[0] = m.mean;
            stats[1] = m.m2;
        }
    }
    __syncthreads();
    if (!*gathered) {
        // Some workgroup of this group has not published in time (it is not
        // resident yet, e.g. while other kernels hold the CUs).  Recompute
        // every part's moments here with the same loads, thread mapping and
        // arithmetic its owner uses, and merge them in the same order: the
        // statistics come out bit-identical, and the kernel never depends on
        // co-residency.  (In-place calls never take this path: they are
        // routed to the two-kernel form, since a chunk already normalised in
        // place could not be re-read.)
        Moments acc{0.f, 0.f, 0.f};
        const int lane = threadIdx.x & (kWave - 1);
        for (int q = 0; q < p.ex.parts; ++q) {
            c.load(p, ng, q);
            const Moments mq = moments_block<kNT / kWave>(c.moments(p, q), lds);
            if ((q & (kWave - 1)) == lane) acc = chan(acc, mq);
        }
        if (threadIdx.x < kWave) {
            acc = moments_wave(acc);
            if (threadIdx.x == 0) {
                stats[0] = acc.mean;
                stats[1] = acc.m2;
                ex_count_give_up(p.ex);
            }
        }
        c.load(p, ng, part);
        __syncthreads();
    }
    // This workgroup is done reading its group's slots: count it out before
    // the stores, so the atomic's round trip overlaps them.
    const bool leaves = p.ex.parts > 1 && threadIdx.x == 0;
    unsigned before = 0;
    if (leaves) before = ex_depart(p.ex, ng);
    c.normalise_store(p, ng, part, stats[0], stats[1]);
    if (leaves) ex_leave(p.ex, ng, before);
}

template <class T, class A, bool VECTOR, bool NHWC>
__global__ __launch_bounds__(kNT) void gn_fused(GNParams p) {
    using C = Chunk<T, VECTOR, NHWC>;
    __shared__ Moments lds[kNT / kWave];
    __shared__ float stats[2];
    __shared__ int gathered;
    int64_t ng;
    int part;
    block_chunk(p, blockIdx.x, &ng, &part);
    const int g = (int)(ng % p.groups);

    C c;
    // Non-temporal for NCHW, where each chunk is read once; channels last
    // keeps the lines in L2, where the workgroups of the neighbouring groups
    // that share them read them too.
    c.template load<!NHWC>(p, ng, part);
    c.template load_affine<A>(p, part, g);
    const Moments m = moments_block<kNT / kWave>(c.moments(p, part), lds);
    if (p.ex.parts > 1 && threadIdx.x == 0) ex_publish(p.ex, ng, part, encode(m));
    settle(p, c, ng, part, m, lds, stats, &gathered);
}

template <class T, bool VECTOR, bool NHWC>
__global__ __launch_bounds__(kNT) void gn_stats(GNParams p) {
    using C = Chunk<T, VECTOR, NHWC>;
    __shared__ Moments lds[kNT / kWave];
    int64_t ng;
    int part;
    block_chunk(p, blockIdx.x, &ng, &part);
    C c;
    c.load(p, ng, part);
    Moments m = moments_block<kNT / kWave>(c.moments(p, part), lds);
    if (threadIdx.x == 0) ex_publish(p.ex, ng, part, encode(m));
}

template <class T, class A, bool VECTOR, bool NHWC>
__global__ __launch_bounds__(kNT) void gn_apply(GNParams p) {
    using C = Chunk<T, VECTOR, NHWC>;
    __shared__ float stats[2];
    int64_t ng;
    int part;
    block_chunk(p, blockIdx.x, &ng, &part);
    const int g = (int)(ng % p.groups);
    // Chunk and affine loads first, so they are in flight while wave 0
    // gathers the statistics.
    C c;
    c.load(p, ng, part);
    c.template load_affine<A>(p, part, g);
    if (threadIdx.x < kWave) {
        bool ok;
        Moments m = gather_parts(p, ng, C::CH, false, &ok);
        if (threadIdx.x == 0) ex_release(p.ex, ng);
        if (threadIdx.x == 0) {
            stats[0] = m.mean;
            stats[1] = m.m2;
        }
    }
    __syncthreads();
    c.normalise_store(p, ng, part, stats[0], stats[1]);
}

// --------------------------------------------------------------------------
// gn_pipe: the fused kernel for dense NCHW 16-bit tensors whose spatial
// size is a multiple of 2048.  A workgroup is four data waves and one
// exchange wave and carries R chunks of 2048 * NV elements, one per round;
// round r holds whole groups only (groups r * per_round ...), so a round's
// exchange never waits on a later round.  The data waves issue the loads of
// every round at once and hold the chunks in registers as raw 16-bit pairs.
// The exchange wave does all the cross-workgroup work (publish, poll, merge,
// affine, departure): loads return in issue order per wave, so a poll issued
// by a wave that still has chunk loads outstanding would wait for them; this
// wave has none.  Against gn_fused on the SD3.5 VAE block (12.1 us per call)
// this form runs 8.3 us: its per-element work is four VALU operations
// instead of about ten, and its merges have no divergent branches.
//
// Moments of a data wave: raw sums S1 = sum x and S2 = sum x^2, each pair of
// 16-bit values folded by one v_dot2 (their products are exact in fp32),
// reduced over the wave's lanes; S1 in double from the lanes' fp32 sums on,
// and the means merged in double.  The mean enters every output as an
// absolute error (x - mean) * a: one fp32 rounding of a mean near 0.3 is
// already 1.5e-8, 1 to 3 bf16 units in the last place of outputs just above
// 2^-19, whereas the lanes' rounding errors average out and the double sums
// keep the group mean within about 1e-10.  The output is then
// (x - hi) * a + (b - lo * a) with the mean split as hi + lo in fp32.  M2 = S2 - S1^2/n
// cancels when the mean is large against the spread, so it is used only when
// 64 * M2 >= S2 (mean^2 <= 63 var over the wave's values), where its
// relative error stays below 2^-12 (a shift of at most 2^-13 of the output
// before rounding to 16 bits); otherwise the wave recomputes M2 exactly:
// per-lane squared deviations from the lane's mean, merged over lanes.  All
// merges are of equal counts, where the Chan et al. update is
// M2 = Ma + Mb + (mb - ma)^2 * n / 2 for n values per side; operands are
// ordered by lane (or wave, or part), so both lanes of a butterfly pair get
// identical bits and the result depends on that order alone.
constexpr int kPipeDataWaves = 4;
constexpr int kPipeNT = (kPipeDataWaves + 1) * kWave;

struct PipeParams {
    const void* x;
    void* y;
    const void* w;
    const void* b;
    Exchange ex;                 // one unit per (sample, group), ex.parts chunks each
    int64_t group_elems;         // (c/G) * spatial
    int64_t spatial;             // a multiple of 2048: every 16-byte slot row lies in one channel
    int32_t cpg;                 // channels per group
    int32_t groups;              // G
    int32_t groups_total;        // n * G
    int32_t per_round;           // groups per round
    int32_t stagger_from;        // first workgroup whose loads wait stagger_ticks (INT32_MAX: none)
    uint32_t stagger_ticks;      // 100 MHz ticks of s_memrealtime
    int32_t force_recompute;     // gn_split only, tests: recompute the parts as if a wait had run out
    float eps;
};

// Moments of a set of values: the mean in double, M2 in float.
struct PipeMoments {
    double mean;
    float m2;
};

// a.x * b.x + a.y * b.y + c on two packed 16-bit values.
__device__ __forceinline__ float dot2(BF16, uint32_t a, uint32_t b, float c) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a), __builtin_bit_cast(bf16x2, b), c, false);
}
__device__ __forceinline__ float dot2(F16, uint32_t a, uint32_t b, float c) {
    return __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2, a), __builtin_bit_cast(f16x2, b), c, false);
}
__device__ __forceinline__ uint32_t ones2(BF16) { return 0x3F803F80u; }
__device__ __forceinline__ uint32_t ones2(F16) { return 0x3C003C00u; }

// Butterfly partner of a double (both halves moved by the same DPP /
// permlane pattern).
template <int S>
__device__ __forceinline__ double partner_f64(double v) {
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const float lo = partner<S>(__uint_as_float((uint32_t)u));
    const float hi = partner<S>(__uint_as_float((uint32_t)(u >> 32)));
    return __builtin_bit_cast(double, (uint64_t)__float_as_uint(lo) | ((uint64_t)__float_as_uint(hi) << 32));
}

// Equal-count merge of a and b (a first), n values each.
__device__ __forceinline__ PipeMoments merge_equal(PipeMoments a, PipeMoments b, float n) {
#pragma clang fp contract(off)
    PipeMoments m;
    m.mean = (a.mean + b.mean) * 0.5;
    const float d = (float)(b.mean - a.mean);
    m.m2 = fmaf(d * d, 0.5f * n, a.m2 + b.m2);
    return m;
}

// Butterfly step S over moments, the lower lane of each pair first.
template <int S>
__device__ __forceinline__ PipeMoments pipe_step(PipeMoments m, float n) {
    const PipeMoments o{partner_f64<S>(m.mean), partner<S>(m.m2)};
    const bool lower = (__lane_id() & (1 << S)) == 0;
    return merge_equal(lower ? m : o, lower ? o : m, n);
}

// Moments of one wave's values: lane l holds NV 16-byte words of 16-bit
// values.  Uniform across the wave.
template <class T, int NV>
__device__ __forceinline__ PipeMoments wave_moments(const u32x4 (&v)[NV]) {
#pragma clang fp contract(off)
    constexpr float kLane = (float)(NV * 8);
    constexpr double kWaveN = (double)kLane * kWave;
    float s1a = 0.f, s1b = 0.f, s2a = 0.f, s2b = 0.f;
#pragma unroll
    for (int j = 0; j < NV; ++j) {
#pragma unroll
        for (int i = 0; i < 4; i += 2) {
            s1a = dot2(T{}, v[j][i], ones2(T{}), s1a);
            s2a = dot2(T{}, v[j][i], v[j][i], s2a);
            s1b = dot2(T{}, v[j][i + 1], ones2(T{}), s1b);
            s2b = dot2(T{}, v[j][i + 1], v[j][i + 1], s2b);
        }
    }
    const float lane_s1 = s1a + s1b;
    // The wave's sum in double (the addition is commutative, so both lanes
    // of a pair get the same bits).
    double s1 = (double)lane_s1;
    s1 += partner_f64<0>(s1);
    s1 += partner_f64<1>(s1);
    s1 += partner_f64<2>(s1);
    s1 += partner_f64<3>(s1);
    s1 += partner_f64<4>(s1);
    s1 += partner_f64<5>(s1);
    const float s2 = group_reduce<kWave>(s2a + s2b, OpSum{});
    PipeMoments m;
    m.mean = s1 * (1.0 / kWaveN);
    m.m2 = s2 - (float)(s1 * m.mean);
    if (__builtin_expect(m.m2 * 64.f >= s2, 1)) return m;
    // Exact M2: per-lane squared deviations from the lane's mean (values
    // widened again here, so no register copy of them is held), merged over
    // the lanes; the wave's mean stays.
    const float mt = lane_s1 * (1.f / kLane);
    float mt2 = 0.f;
#pragma unroll
    for (int j = 0; j < NV; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            float lo, hi;
            unpack2(T{}, v[j][i], lo, hi);
            const float dl = lo - mt, dh = hi - mt;
            mt2 = fmaf(dl, dl, mt2);
            mt2 = fmaf(dh, dh, mt2);
        }
    PipeMoments t{(double)mt, mt2};
    t = pipe_step<0>(t, kLane);
    t = pipe_step<1>(t, 2.f * kLane);
    t = pipe_step<2>(t, 4.f * kLane);
    t = pipe_step<3>(t, 8.f * kLane);
    t = pipe_step<4>(t, 16.f * kLane);
    t = pipe_step<5>(t, 32.f * kLane);
    m.m2 = t.m2;
    return m;
}

// Stores of a chunk's output, non-temporal and device-scope (write-through):
// the output lines go on to HBM as they are written instead of waiting in L2
// for the end-of-kernel write-back.  A 16 MiB output fits in the L2s, and
// with plain non-temporal stores the write-back of all of it ran after the
// last workgroup had finished (SD3.5 VAE block 8.59 -> 8.26 us per call).
// Written as raw buffer stores, whose cache-policy operand takes these bits,
// over a descriptor that spans exactly the chunk (stores outside a buffer's
// range are dropped, never performed); the compiler sees them as stores and
// keeps the wait states a 16-byte store needs before its data registers are
// reused.
constexpr int kCpolNtSc1 = 2 | 16;           // nt | sc1
constexpr int kRawBufferWord3 = 0x00020000;  // 32-bit data format, raw access
__device__ __forceinline__ __amdgpu_buffer_rsrc_t chunk_buffer(char* base, int64_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(base, 0, (int)bytes, kRawBufferWord3);
}
__device__ __forceinline__ void store16_through(__amdgpu_buffer_rsrc_t r, int offset, u32x4 v) {
    __builtin_amdgcn_raw_buffer_store_b128(v, r, offset, 0, kCpolNtSc1);
}

// Loads of chunk (ng, part) for virtual thread t (0..255): slot j holds the
// 16 bytes at element (j * 256 + t) * 8 of the chunk.
template <int NV>
__device__ __forceinline__ void pipe_load(const PipeParams& p, int64_t ng, int part, int t, u32x4 (&v)[NV]) {
    constexpr int64_t CH = (int64_t)kPipeDataWaves * kWave * NV * 8;
    const char* base = static_cast<const char*>(p.x) + (ng * p.group_elems + part * CH) * 2;
#pragma unroll
    for (int j = 0; j < NV; ++j) v[j] = load16<true>(base + ((int64_t)j * 256 + t) * 16);
}

// Moments of a whole chunk from its four wave partials, in a fixed tree.
template <int NV>
__device__ __forceinline__ PipeMoments chunk_moments(const PipeMoments (&w)[kPipeDataWaves]) {
    constexpr float kWaveN = (float)(NV * 8 * kWave);
    return merge_equal(merge_equal(w[0], w[1], kWaveN), merge_equal(w[2], w[3], kWaveN), 2.f * kWaveN);
}

// A part's moments as one published word, never 0 (the value of an empty
// slot), written with one single-copy-atomic store: the part's mean rounded
// to fp32 in the low half, M2 in the high half with its sign bit (M2 >= 0)
// forced on.  M2 keeps full fp32 precision: near y = 0 the output is the
// difference of (x - mean) * a and -b, so a relative error e of the rstd
// inside a shows as an absolute error |b| * e there (a 15-bit M2 measured
// 1e-6 of it).  The mean loses at most half an fp32 unit per part; the
// group mean is the double average of the P part means.
__device__ __forceinline__ uint64_t pipe_encode(PipeMoments m) {
    return (uint64_t)__float_as_uint((float)m.mean) |
           ((uint64_t)(__float_as_uint(fmaxf(m.m2, 0.f)) | 0x80000000u) << 32);
}
__device__ __forceinline__ PipeMoments pipe_decode(uint64_t w) {
    return PipeMoments{(double)__uint_as_float((uint32_t)w), __uint_as_float((uint32_t)(w >> 32) & 0x7fffffffu)};
}

// The group's statistics for the exchange wave: every part's published
// word (lane q polls part q's), merged in
// part order (P a power of two <= 64).  Without all parts published in time,
// the wave recomputes every part's moments with the data waves' loads, lane
// mapping and arithmetic, so the result is bit-identical either way.
template <class T, int NV>
__device__ __forceinline__ PipeMoments pipe_gather(const PipeParams& p, int64_t ng) {
    constexpr float kChunkN = (float)(NV * 8 * kWave * kPipeDataWaves);
    const int lane = threadIdx.x & (kWave - 1);
    const int P = p.ex.parts;
    const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
    PipeMoments m{0.0, 0.f};
    bool ok = true;
    if (lane < P) {
        uint64_t* at = ex_slot(p.ex, ng, lane);
        uint64_t w = __hip_atomic_load(at, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        while (w == 0) {
            if (__builtin_amdgcn_s_memrealtime() - t0 > p.ex.wait_ticks) break;
            w = __hip_atomic_load(at, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        ok = w != 0;
        m = pipe_decode(w);
    }
    if (!__all(ok)) {
        for (int q = 0; q < P; ++q) {
            PipeMoments w[kPipeDataWaves];
#pragma unroll
            for (int k = 0; k < kPipeDataWaves; ++k) {
                u32x4 v[NV];
                pipe_load<NV>(p, ng, q, k * kWave + lane, v);
                w[k] = wave_moments<T, NV>(v);
            }
            // Through the same encoding a published word takes, so the
            // statistics match the normal path bit for bit.
            const PipeMoments c = pipe_decode(pipe_encode(chunk_moments<NV>(w)));
            if (lane == q) m = c;
        }
        if (lane == 0) ex_count_give_up(p.ex);
    }
    // Merge over P lanes (P = 2^k): the first k butterfly steps.
    float n = kChunkN;
#define KF_STEP(S)                    \
    if ((2 << S) <= P) {              \
        m = pipe_step<S>(m, n);       \
        n *= 2.f;                     \
    }
    KF_STEP(0) KF_STEP(1) KF_STEP(2) KF_STEP(3) KF_STEP(4) KF_STEP(5)
#undef KF_STEP
    const uint64_t u = __builtin_bit_cast(uint64_t, m.mean);
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)u), hi = __builtin_amdgcn_readfirstlane((uint32_t)(u >> 32));
    return PipeMoments{__builtin_bit_cast(double, (uint64_t)lo | ((uint64_t)hi << 32)), uniform0(m.m2)};
}

// The (group, part) chunk workgroup b handles in round r: group-major, a
// group's parts on consecutive workgroups (so spread over the XCDs, which
// take workgroups in turn), the earliest groups dispatched first.  Placing
// all parts of a group on one XCD measured 8.41 against 8.29 us on the
// SD3.5 VAE block.
__device__ __forceinline__ void pipe_chunk(const PipeParams& p, int b, int r, int64_t* ng, int* part) {
    const int P = p.ex.parts;
    *ng = (int64_t)r * p.per_round + b / P;
    *part = b - (b / P) * P;
}

template <class T, class A, int NV, int R>
__global__ __launch_bounds__(kPipeNT) void gn_pipe(PipeParams p) {
    constexpr int64_t CH = (int64_t)kPipeDataWaves * kWave * NV * 8;
    __shared__ PipeMoments part_lds[R][kPipeDataWaves];
    __shared__ float stats_lds[R][NV][2];  // per slot: a = rstd * w[c], c = b[c] - lo * a
    __shared__ float mean_lds[R];          // hi of the group mean
    const int wave = threadIdx.x / kWave;
    const int lane = threadIdx.x & (kWave - 1);

    if (wave < kPipeDataWaves) {
        // Staggered issue: the second half of a grid with two or more
        // workgroups per CU issues its loads a fixed time after it starts.
        // The first half's groups then complete sooner and store while the
        // second half still loads, as a copy overlaps its reads and writes.
        if ((int)blockIdx.x >= p.stagger_from) {
            const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
            while (__builtin_amdgcn_s_memrealtime() - t0 < p.stagger_ticks) __builtin_amdgcn_s_sleep(1);
        }
        u32x4 v[R][NV];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            int64_t ng;
            int part;
            pipe_chunk(p, blockIdx.x, r, &ng, &part);
            pipe_load<NV>(p, ng < p.groups_total ? ng : p.groups_total - 1, part, threadIdx.x, v[r]);
        }
#pragma unroll
        for (int r = 0; r < R; ++r) {
            int64_t ng;
            int part;
            pipe_chunk(p, blockIdx.x, r, &ng, &part);
            const bool live = ng < p.groups_total;
            if (live) {
                const PipeMoments m = wave_moments<T, NV>(v[r]);
                if (lane == 0) part_lds[r][wave] = m;
            }
            __syncthreads();  // partials of round r in LDS
            __syncthreads();  // statistics of round r in LDS
            if (live) {
                // y = (x - hi) * a + (b - lo * a): x - hi is exact wherever
                // the output is near zero (x within a factor 2 of hi).
                const __amdgpu_buffer_rsrc_t out =
                    chunk_buffer(static_cast<char*>(p.y) + (ng * p.group_elems + part * CH) * 2, CH * 2);
                const float mu = mean_lds[r];
#pragma unroll
                for (int j = 0; j < NV; ++j) {
                    const float a = stats_lds[r][j][0], c = stats_lds[r][j][1];
                    u32x4 o;
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        float lo, hi;
                        unpack2(T{}, v[r][j][i], lo, hi);
                        o[i] = pack2(T{}, fmaf(lo - mu, a, c), fmaf(hi - mu, a, c));
                    }
                    store16_through(out, (j * 256 + (int)threadIdx.x) * 16, o);
                }
            }
        }
    } else {
        // Affine of each round's slot channels (lane j: slot j), loaded
        // first: nothing waits on them until the statistics are known.
        const bool hw = p.w != nullptr, hb = p.b != nullptr;
        const void* ws = hw ? p.w : affine_identity<A>();
        const void* bs = hb ? p.b : affine_identity<A>();
        float wv[R], bv[R];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            int64_t ng;
            int part;
            pipe_chunk(p, blockIdx.x, r, &ng, &part);
            if (ng >= p.groups_total) ng = p.groups_total - 1;
            const int j = lane < NV ? lane : 0;
            const int64_t c = (ng % p.groups) * p.cpg + (part * CH + (int64_t)j * 2048) / p.spatial;
            wv[r] = load1<A>(ws, hw ? c : 0);
            bv[r] = load1<A>(bs, hb ? c : 1);
        }
#pragma unroll
        for (int r = 0; r < R; ++r) {
            int64_t ng;
            int part;
            pipe_chunk(p, blockIdx.x, r, &ng, &part);
            const bool live = ng < p.groups_total;
            __syncthreads();  // partials of round r in LDS
            unsigned before = 0;
            if (live) {
                PipeMoments w[kPipeDataWaves];
#pragma unroll
                for (int k = 0; k < kPipeDataWaves; ++k) w[k] = part_lds[r][k];
                const PipeMoments mine = chunk_moments<NV>(w);
                if (lane == 0) ex_publish(p.ex, ng, part, pipe_encode(mine));
                const PipeMoments g = pipe_gather<T, NV>(p, ng);
                // Done reading the group's slots: count this workgroup out
                // now, so the atomic's round trip overlaps the rest.
                if (lane == 0) before = ex_depart(p.ex, ng);
                const float rstd = 1.f / sqrtf(g.m2 / (float)p.group_elems + p.eps);
                const float hi = (float)g.mean, lo = (float)(g.mean - (double)hi);
                if (lane < NV) {
                    const float a = rstd * wv[r];
                    stats_lds[r][lane][0] = a;
                    stats_lds[r][lane][1] = bv[r] - lo * a;
                }
                if (lane == 0) mean_lds[r] = hi;
            }
            __syncthreads();  // statistics of round r in LDS
            if (live && lane == 0) ex_leave(p.ex, ng, before);
        }
    }
}

// --------------------------------------------------------------------------
// gn_split: GroupNorm in two launches for dense NCHW 16-bit tensors whose
// one-launch grid cannot be resident (the SD3.5 VAE decoder's full-size
// blocks, e.g. [1, 128, 1024, 1024]: 256 MiB, no register file holds it), in
// gn_pipe's arithmetic.  gn_split_stats reads each 16384-element chunk once,
// folds its moments with v_dot2 and publishes them; the last workgroup of a
// group to arrive (a per-group counter) merges the group's parts in part
// order and writes the group's mean (double) and M2 into the second 128-byte
// line of the group's 256-byte counter stride (the counter is bytes 0-3 of
// the first, so the second launch's departure atomics do not contend with
// its reads of the statistics; 194 against 137 us with both in one line on
// [1, 128, 1024, 1024]), never over a part's slot, which a publish still in
// flight could overwrite.
// gn_split_apply re-reads each chunk and normalises it with those
// statistics; its last workgroup of a group returns the group's slots,
// statistics words and counter to zero.  One read more than gn_pipe, but
// both passes stream (45 + 90 us on [1, 128, 1024, 1024], where the moments
// pass of the general two-kernel form, about ten VALU operations per
// element, ran 71 us: a read at 3.8 TB/s).

// a + b for moments of na and nb values (a first).
__device__ __forceinline__ PipeMoments merge_counts(PipeMoments a, PipeMoments b, float na, float nb) {
#pragma clang fp contract(off)
    const float nt = na + nb;
    PipeMoments m;
    m.mean = a.mean + (b.mean - a.mean) * ((double)nb / (double)nt);
    const float d = (float)(b.mean - a.mean);
    m.m2 = fmaf(d * d, na * (nb / nt), a.m2 + b.m2);
    return m;
}

// The P parts of group ng merged in part order by one wave: lane l folds
// parts l, l + 64, l + 128, ... in that order, then the lane butterfly over
// min(P, 64) lanes (P a power of two).  Every part has been published (the
// caller is the group's last arrival), so the bounded wait only guards the
// memory model; if a part is still unseen after it, the wave recomputes
// every part from x with its owner's loads and arithmetic, bit for bit.
template <class T, int NV>
__device__ PipeMoments split_gather(const PipeParams& p, int64_t ng) {
    constexpr float kChunkN = (float)(NV * 8 * kWave * kPipeDataWaves);
    constexpr int kBatch = 4;  // slot loads in flight per lane
    const int lane = threadIdx.x & (kWave - 1);
    const int P = p.ex.parts;
    const int per = P > kWave ? P / kWave : 1;
    const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
    PipeMoments acc{0.0, 0.f};
    bool ok = true;
    for (int i0 = 0; i0 < per; i0 += kBatch) {
        uint64_t w[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int q = lane + (i0 + u) * kWave;
            w[u] = (i0 + u < per && q < P) ? __hip_atomic_load(ex_slot(p.ex, ng, q), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 1;
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int i = i0 + u;
            const int q = lane + i * kWave;
            if (i < per && q < P) {
                if (w[u] == 0) w[u] = ex_poll(p.ex, ng, q, t0, true);
                ok = ok && w[u] != 0;
                const PipeMoments mi = pipe_decode(w[u]);
                acc = i == 0 ? mi : merge_counts(acc, mi, (float)i * kChunkN, kChunkN);
            }
        }
    }
    if (!__all(ok) || p.force_recompute) {
        acc = PipeMoments{0.0, 0.f};
        for (int q = 0; q < P; ++q) {
            PipeMoments w[kPipeDataWaves];
#pragma unroll
            for (int k = 0; k < kPipeDataWaves; ++k) {
                u32x4 v[NV];
                pipe_load<NV>(p, ng, q, k * kWave + lane, v);
                w[k] = wave_moments<T, NV>(v);
            }
            const PipeMoments c = pipe_decode(pipe_encode(chunk_moments<NV>(w)));
            const int i = q / kWave;
            if ((q & (kWave - 1)) == lane) acc = i == 0 ? c : merge_counts(acc, c, (float)i * kChunkN, kChunkN);
        }
        if (lane == 0) ex_count_give_up(p.ex);
    }
    float n = (float)per * kChunkN;
    const int lanes = P < kWave ? P : kWave;
#define KF_STEP(S)                    \
    if ((2 << S) <= lanes) {          \
        acc = pipe_step<S>(acc, n);   \
        n *= 2.f;                     \
    }
    KF_STEP(0) KF_STEP(1) KF_STEP(2) KF_STEP(3) KF_STEP(4) KF_STEP(5)
#undef KF_STEP
    const uint64_t u = __builtin_bit_cast(uint64_t, acc.mean);
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)u), hi = __builtin_amdgcn_readfirstlane((uint32_t)(u >> 32));
    return PipeMoments{__builtin_bit_cast(double, (uint64_t)lo | ((uint64_t)hi << 32)), uniform0(acc.m2)};
}

// The group's statistics words: the mean (double bits) and M2 (fp32 bits),
// at byte 128 of the group's 256-byte counter stride.
__device__ __forceinline__ uint64_t* split_stats(const PipeParams& p, int64_t ng) {
    return reinterpret_cast<uint64_t*>(reinterpret_cast<char*>(ex_counter(p.ex, ng)) + 128);
}

__device__ __forceinline__ void split_chunk(const PipeParams& p, int b, int64_t* ng, int* part) {
    const int P = p.ex.parts;
    *ng = b / P;
    *part = b - (b / P) * P;
}

template <class T, int NV>
__global__ __launch_bounds__(kPipeDataWaves * kWave) void gn_split_stats(PipeParams p) {
    __shared__ PipeMoments part_lds[kPipeDataWaves];
    __shared__ unsigned before_lds;
    const int wave = threadIdx.x / kWave;
    const int lane = threadIdx.x & (kWave - 1);
    int64_t ng;
    int part;
    split_chunk(p, blockIdx.x, &ng, &part);
    u32x4 v[NV];
    pipe_load<NV>(p, ng, part, threadIdx.x, v);
    const PipeMoments m = wave_moments<T, NV>(v);
    if (lane == 0) part_lds[wave] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
        PipeMoments w[kPipeDataWaves];
#pragma unroll
        for (int k = 0; k < kPipeDataWaves; ++k) w[k] = part_lds[k];
        ex_publish(p.ex, ng, part, pipe_encode(chunk_moments<NV>(w)));
        // Relaxed, like every exchange access here: an agent-scope release
        // or acquire writes back or invalidates the L2, which thousands of
        // workgroups cannot afford.  The last arrival may see the count
        // before some published word; it polls for the words (self-flagged).
        before_lds = ex_depart(p.ex, ng);
    }
    __syncthreads();
    if (wave != 0 || before_lds != (unsigned)p.ex.parts - 1) return;
    // The group's last arrival: every part is published.
    const PipeMoments g = split_gather<T, NV>(p, ng);
    if (lane == 0) {
        uint64_t* r = split_stats(p, ng);
        __hip_atomic_store(r, __builtin_bit_cast(uint64_t, g.mean), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(r + 1, (uint64_t)__float_as_uint(g.m2), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(ex_counter(p.ex, ng), 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

template <class T, class A, int NV>
__global__ __launch_bounds__(kPipeDataWaves * kWave) void gn_split_apply(PipeParams p) {
    constexpr int64_t CH = (int64_t)kPipeDataWaves * kWave * NV * 8;
    __shared__ float stats_lds[NV][2];  // per slot: a = rstd * w[c], c = b[c] - lo * a
    __shared__ float mean_lds;          // hi of the group mean
    const int lane = threadIdx.x & (kWave - 1);
    int64_t ng;
    int part;
    split_chunk(p, blockIdx.x, &ng, &part);
    u32x4 v[NV];
    pipe_load<NV>(p, ng, part, threadIdx.x, v);
    if (threadIdx.x < kWave) {
        // Lane j: the affine of slot j's channel, and the group statistics
        // gn_split_stats left beside the counter (visible: an earlier launch
        // on the same stream wrote them).
        const bool hw = p.w != nullptr, hb = p.b != nullptr;
        const void* ws = hw ? p.w : affine_identity<A>();
        const void* bs = hb ? p.b : affine_identity<A>();
        const int j = lane < NV ? lane : 0;
        const int64_t c = (ng % p.groups) * p.cpg + (part * CH + (int64_t)j * 2048) / p.spatial;
        const float wv = load1<A>(ws, hw ? c : 0);
        const float bv = load1<A>(bs, hb ? c : 1);
        uint64_t* r = split_stats(p, ng);
        const uint64_t mw = __hip_atomic_load(r, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const uint64_t vw = __hip_atomic_load(r + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const double mean = __builtin_bit_cast(double, mw);
        const float m2 = __uint_as_float((uint32_t)vw);
        const float rstd = 1.f / sqrtf(m2 / (float)p.group_elems + p.eps);
        const float hi = (float)mean, lo = (float)(mean - (double)hi);
        if (lane < NV) {
            const float a = rstd * wv;
            stats_lds[lane][0] = a;
            stats_lds[lane][1] = bv - lo * a;
        }
        if (lane == 0) mean_lds = hi;
        // Done reading the group's statistics: rstd consumes both loads, so
        // they have returned before the departure count (relaxed; the empty
        // asm keeps the count after them).  The last workgroup of the group
        // empties its slots and counter.
        __asm__ volatile("" : : "v"(rstd), "v"(lo) : "memory");
        unsigned before = 0;
        if (lane == 0) before = ex_depart(p.ex, ng);
        before = __builtin_amdgcn_readfirstlane(before);
        if (before == (unsigned)p.ex.parts - 1) {
            for (int q = lane; q < p.ex.parts; q += kWave)
                __hip_atomic_store(ex_slot(p.ex, ng, q), (uint64_t)0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (lane < 2) __hip_atomic_store(r + lane, (uint64_t)0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (lane == 0) __hip_atomic_store(ex_counter(p.ex, ng), 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
    __syncthreads();
    const __amdgpu_buffer_rsrc_t out = chunk_buffer(static_cast<char*>(p.y) + (ng * p.group_elems + part * CH) * 2, CH * 2);
    const float mu = mean_lds;
#pragma unroll
    for (int j = 0; j < NV; ++j) {
        const float a = stats_lds[j][0], c = stats_lds[j][1];
        u32x4 o;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            float x0, x1;
            unpack2(T{}, v[j][i], x0, x1);
            o[i] = pack2(T{}, fmaf(x0 - mu, a, c), fmaf(x1 - mu, a, c));
        }
        store16_through(out, (j * 256 + (int)threadIdx.x) * 16, o);
    }
}

// --------------------------------------------------------------------------
// gn_pipe_cl: gn_pipe for dense channels-last 16-bit tensors [n, hw, c]
// with c a multiple of 64 and cpg in {8, 16, 32, 64}.  A tile is 64 adjacent
// channels (one 128-byte line per pixel, Q = 64 / cpg whole groups) of 256
// consecutive pixels of one sample; a workgroup owns one tile, so every
// line it reads or writes is a whole line of its own, and a group splits
// into hw / 256 parts (a power of two, at most 64).  Lane l of a data wave
// holds, in slot j, the 16 bytes of tile channels 8 * (l % 8) .. + 7 at
// pixel j * 32 + wave * 8 + l / 8: each load reads eight whole lines, the
// eight lanes of one line consecutive (with the lanes of a line 8 apart
// instead, the same access pattern as a plain copy took 8.1 against 7.6 us
// on 16 MiB).  A group's lanes are a block of cpg / 8 lanes in each of the
// eight 8-lane rows, so its moments reduce over the block (xor 1, 2, 4) and
// then over the rows (xor 8 by ds_swizzle, 16 and 32 by permlane swaps).
// Workgroups are numbered tile-column-major: the first 64-channel column's
// parts go out first, so its groups finish and store while later columns
// still load (with each column's parts on one XCD, all columns ran side by
// side and none could store before the last loads: 14.6 against 12.6 us on
// the SD3.5 VAE block).  The exchange wave publishes, gathers and merges
// the tile's Q groups together (lane q polls part q of each).  Otherwise as
// gn_pipe: raw 16-bit pairs in registers, v_dot2 sums, double means,
// bit-identical recompute when a wait gives up, write-through stores.
constexpr int kClNV = 8;                               // slots per lane
// Exchange slots of gn_pipe_cl one 128-byte line apart: its 64 parts per
// group would otherwise publish 16 to a line (SD3.5 block in channels last,
// two boxes: 12.65 -> 11.97 us and 12.28 -> 12.00; 2 words apart 12.16 on
// the first; the NCHW gn_pipe, 16 parts per group, gained nothing from it
// and keeps its packed slots).
constexpr int kClSlotStride = 16;
constexpr int kClPixels = kPipeDataWaves * 8 * kClNV;  // pixels per tile: 256

struct PipeClParams {
    const void* x;
    void* y;
    const void* w;
    const void* b;
    Exchange ex;          // one unit per (sample, group), ex.parts tiles each
    int64_t hw;           // pixels per sample
    int32_t c;            // channels, a multiple of 64
    int32_t groups;       // G
    int32_t tiles_total;  // n * c / 64
    float eps;
};

// Partner of a float across lanes X apart (X a power of two): xor 1 and 2
// are quad permutations; 4 is the half-row mirror, a butterfly partner only
// after the xor-1 and xor-2 steps (as every use here is); 8 is a ds_swizzle
// bitmask xor; 16 and 32 the permlane swaps.
template <int X>
__device__ __forceinline__ float xor_partner(float v) {
    if constexpr (X == 1) return partner<0>(v);
    else if constexpr (X == 2) return partner<1>(v);
    else if constexpr (X == 4) return partner<2>(v);
    else if constexpr (X == 8)
        return __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, v), 0x201F));
    else if constexpr (X == 16) return partner<4>(v);
    else return partner<5>(v);
}
template <int X>
__device__ __forceinline__ double xor_partner_f64(double v) {
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const float lo = xor_partner<X>(__uint_as_float((uint32_t)u));
    const float hi = xor_partner<X>(__uint_as_float((uint32_t)(u >> 32)));
    return __builtin_bit_cast(double, (uint64_t)__float_as_uint(lo) | ((uint64_t)__float_as_uint(hi) << 32));
}
template <int X>
__device__ __forceinline__ PipeMoments xor_step(PipeMoments m, float n) {
    const PipeMoments o{xor_partner_f64<X>(m.mean), xor_partner<X>(m.m2)};
    const bool lower = (__lane_id() & X) == 0;
    return merge_equal(lower ? m : o, lower ? o : m, n);
}

// The lane distances a group's lanes are reduced over, in order: its block
// of CPG / 8 lanes, then the eight rows.
template <int CPG, class F>
__device__ __forceinline__ void cl_steps(F&& step) {
    if constexpr (CPG >= 16) step(std::integral_constant<int, 1>{});
    if constexpr (CPG >= 32) step(std::integral_constant<int, 2>{});
    if constexpr (CPG >= 64) step(std::integral_constant<int, 4>{});
    step(std::integral_constant<int, 8>{});
    step(std::integral_constant<int, 16>{});
    step(std::integral_constant<int, 32>{});
}

// Moments of each group's values in one wave (lane l holds kClNV 16-byte
// words of its group's values); every lane gets its group's moments.
template <class T, int CPG>
__device__ __forceinline__ PipeMoments lanes_moments(const u32x4 (&v)[kClNV]) {
#pragma clang fp contract(off)
    constexpr float kLane = (float)(kClNV * 8);
    constexpr double kGroupN = (double)kLane * CPG;  // CPG lanes per group
    float s1a = 0.f, s1b = 0.f, s2a = 0.f, s2b = 0.f;
#pragma unroll
    for (int j = 0; j < kClNV; ++j) {
#pragma unroll
        for (int i = 0; i < 4; i += 2) {
            s1a = dot2(T{}, v[j][i], ones2(T{}), s1a);
            s2a = dot2(T{}, v[j][i], v[j][i], s2a);
            s1b = dot2(T{}, v[j][i + 1], ones2(T{}), s1b);
            s2b = dot2(T{}, v[j][i + 1], v[j][i + 1], s2b);
        }
    }
    const float lane_s1 = s1a + s1b;
    double s1 = (double)lane_s1;
    float s2 = s2a + s2b;
    cl_steps<CPG>([&](auto X) {
        s1 += xor_partner_f64<decltype(X)::value>(s1);
        s2 += xor_partner<decltype(X)::value>(s2);
    });
    PipeMoments m;
    m.mean = s1 * (1.0 / kGroupN);
    m.m2 = s2 - (float)(s1 * m.mean);
    const bool fast = m.m2 * 64.f >= s2;
    if (__builtin_expect(__all(fast), 1)) return m;
    // Exact M2 for the groups that need it, as in wave_moments (computed by
    // the whole wave, whose exchanges need every lane).
    const float mt = lane_s1 * (1.f / kLane);
    float mt2 = 0.f;
#pragma unroll
    for (int j = 0; j < kClNV; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            float lo, hi;
            unpack2(T{}, v[j][i], lo, hi);
            const float dl = lo - mt, dh = hi - mt;
            mt2 = fmaf(dl, dl, mt2);
            mt2 = fmaf(dh, dh, mt2);
        }
    PipeMoments t{(double)mt, mt2};
    float n = kLane;
    cl_steps<CPG>([&](auto X) {
        t = xor_step<decltype(X)::value>(t, n);
        n *= 2.f;
    });
    if (!fast) m.m2 = t.m2;
    return m;
}

// The (tile, part) that workgroup b handles: tile-column-major.
// Tile indices fit in 32 bits (tiles_total does), so these divide in 32
// bits (no measurable change on the SD3.5 block: the exchange, not this
// arithmetic, bounds it).
__device__ __forceinline__ void cl_tile(const PipeClParams& p, int b, int* tile, int* part) {
    const int P = p.ex.parts;
    *tile = b / P;
    *part = b - (b / P) * P;
}

// Element index of the first element of part `part` of tile `tile`.
__device__ __forceinline__ int64_t cl_first(const PipeClParams& p, int tile, int part) {
    const int cols = p.c / 64;
    const int n = tile / cols;
    const int col = tile - n * cols;
    return ((int64_t)n * p.hw + (int64_t)part * kClPixels) * p.c + col * 64;
}

// Loads of a tile part for virtual thread t (0..255).
__device__ __forceinline__ void cl_load(const PipeClParams& p, int64_t first, int t, u32x4 (&v)[kClNV]) {
    const char* base = static_cast<const char*>(p.x) + first * 2;
    const int wave = t / kWave, lane = t & (kWave - 1);
#pragma unroll
    for (int j = 0; j < kClNV; ++j) {
        const int64_t px = j * 32 + wave * 8 + (lane >> 3);
        v[j] = load16<true>(base + (px * p.c + (lane & 7) * 8) * 2);
    }
}

// A tile part's moments of group k (0..Q-1) from the four waves' partials.
template <int CPG>
__device__ __forceinline__ PipeMoments cl_part_moments(const PipeMoments (&w)[kPipeDataWaves]) {
    constexpr float kWaveN = (float)(CPG * kClNV * 8);
    return merge_equal(merge_equal(w[0], w[1], kWaveN), merge_equal(w[2], w[3], kWaveN), 2.f * kWaveN);
}

template <class T, class A, int CPG>
__global__ __launch_bounds__(kPipeNT) void gn_pipe_cl(PipeClParams p) {
    constexpr int Q = 64 / CPG;  // groups per tile
    __shared__ PipeMoments part_lds[kPipeDataWaves][Q];
    __shared__ float gstat[Q][3];  // per group: hi and lo of the mean, rstd
    const int wave = threadIdx.x / kWave;
    const int lane = threadIdx.x & (kWave - 1);
    int tile;
    int part;
    cl_tile(p, blockIdx.x, &tile, &part);
    const int64_t first = cl_first(p, tile, part);
    const int cols = p.c / 64;
    const int64_t n = tile / cols;
    const int col = (int)(tile - (int)n * cols);

    if (wave < kPipeDataWaves) {
        u32x4 v[kClNV];
        cl_load(p, first, threadIdx.x, v);
        // The affine of this lane's eight channels, after the tile's loads
        // (nothing waits on it until the statistics are known).
        const bool hw = p.w != nullptr, hb = p.b != nullptr;
        const void* ws = hw ? p.w : affine_identity<A>();
        const void* bs = hb ? p.b : affine_identity<A>();
        const int64_t ch = (int64_t)col * 64 + (lane & 7) * 8;
        float wv[8], bv[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            wv[i] = load1<A>(ws, hw ? ch + i : 0);
            bv[i] = load1<A>(bs, hb ? ch + i : 1);
        }
        constexpr int B = CPG / 8;  // lanes of a group in each 8-lane row
        const PipeMoments m = lanes_moments<T, CPG>(v);
        if (lane < 8 && (lane % B) == 0) part_lds[wave][lane / B] = m;
        __syncthreads();  // partials in LDS
        __syncthreads();  // statistics in LDS
        const int k = (lane & 7) / B;
        const float mu = gstat[k][0], lo = gstat[k][1], rstd = gstat[k][2];
        float a[8], c[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            a[i] = rstd * wv[i];
            c[i] = bv[i] - lo * a[i];
        }
        const int64_t span = ((int64_t)(kClPixels - 1) * p.c + 64) * 2;
        const __amdgpu_buffer_rsrc_t out = chunk_buffer(static_cast<char*>(p.y) + first * 2, span);
#pragma unroll
        for (int j = 0; j < kClNV; ++j) {
            const int64_t px = j * 32 + wave * 8 + (lane >> 3);
            u32x4 o;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                float x0, x1;
                unpack2(T{}, v[j][i], x0, x1);
                o[i] = pack2(T{}, fmaf(x0 - mu, a[2 * i], c[2 * i]), fmaf(x1 - mu, a[2 * i + 1], c[2 * i + 1]));
            }
            store16_through(out, (int)((px * p.c + (lane & 7) * 8) * 2), o);
        }
    } else {
        const int64_t ng0 = n * p.groups + (int64_t)col * Q;  // the tile's first group
        const int P = p.ex.parts;
        __syncthreads();  // partials in LDS
        if (lane < Q) {
            PipeMoments w[kPipeDataWaves];
#pragma unroll
            for (int k = 0; k < kPipeDataWaves; ++k) w[k] = part_lds[k][lane];
            ex_publish(p.ex, ng0 + lane, part, pipe_encode(cl_part_moments<CPG>(w)));
        }
        // Lane q polls part q of every group of the tile, all Q words per
        // pass.
        uint64_t word[Q];
#pragma unroll
        for (int k = 0; k < Q; ++k) word[k] = 0;
        bool ok = true;
        if (lane < P) {
            const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
            for (;;) {
                bool all = true;
#pragma unroll
                for (int k = 0; k < Q; ++k) {
                    word[k] = __hip_atomic_load(ex_slot(p.ex, ng0 + k, lane), __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT);
                    all = all && word[k] != 0;
                }
                if (all) break;
                if (__builtin_amdgcn_s_memrealtime() - t0 > p.ex.wait_ticks) {
                    ok = false;
                    break;
                }
            }
        }
        PipeMoments m[Q];
#pragma unroll
        for (int k = 0; k < Q; ++k) m[k] = pipe_decode(word[k]);
        if (!__all(ok)) {
            // Recompute every part of the tile column with the data waves'
            // loads, lane mapping and arithmetic, through the published
            // encoding, so the statistics match the normal path bit for bit.
            const int64_t first0 = cl_first(p, tile, 0);
            for (int q = 0; q < P; ++q) {
                PipeMoments w[kPipeDataWaves][Q];
#pragma unroll
                for (int kk = 0; kk < kPipeDataWaves; ++kk) {
                    u32x4 v[kClNV];
                    cl_load(p, first0 + (int64_t)q * kClPixels * p.c, kk * kWave + lane, v);
                    const PipeMoments wm = lanes_moments<T, CPG>(v);
                    const uint64_t mb = __builtin_bit_cast(uint64_t, wm.mean);
#pragma unroll
                    for (int k = 0; k < Q; ++k) {
                        const int src = k * (CPG / 8);  // the group's lane in row 0
                        const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)mb, src);
                        const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(mb >> 32), src);
                        w[kk][k].mean = __builtin_bit_cast(double, (uint64_t)lo | ((uint64_t)hi << 32));
                        w[kk][k].m2 = __builtin_bit_cast(
                            float, __builtin_amdgcn_readlane(__builtin_bit_cast(uint32_t, wm.m2), src));
                    }
                }
#pragma unroll
                for (int k = 0; k < Q; ++k) {
                    PipeMoments wk[kPipeDataWaves];
#pragma unroll
                    for (int kk = 0; kk < kPipeDataWaves; ++kk) wk[kk] = w[kk][k];
                    const PipeMoments cq = pipe_decode(pipe_encode(cl_part_moments<CPG>(wk)));
                    if (lane == q) m[k] = cq;
                }
            }
            if (lane == 0) ex_count_give_up(p.ex);
        }
        // Merge each group over P lanes (P = 2^k): the first k butterfly
        // steps, in part order.
        float nn = (float)(kPipeDataWaves * CPG * kClNV * 8);
#define KF_STEP(S)                                                   \
    if ((2 << S) <= P) {                                             \
        _Pragma("unroll") for (int k = 0; k < Q; ++k) m[k] = pipe_step<S>(m[k], nn); \
        nn *= 2.f;                                                   \
    }
        KF_STEP(0) KF_STEP(1) KF_STEP(2) KF_STEP(3) KF_STEP(4) KF_STEP(5)
#undef KF_STEP
        // Lane 0's merge (lanes past P merged empty slots).
#pragma unroll
        for (int k = 0; k < Q; ++k) {
            const uint64_t u = __builtin_bit_cast(uint64_t, m[k].mean);
            const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)u);
            const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(u >> 32));
            m[k] = PipeMoments{__builtin_bit_cast(double, (uint64_t)lo | ((uint64_t)hi << 32)), uniform0(m[k].m2)};
        }
        // Done reading the slots: count this workgroup out of every group
        // of the tile now, so the atomics' round trips overlap the rest.
        unsigned before = 0;
        if (lane < Q) before = ex_depart(p.ex, ng0 + lane);
        const float group_n = (float)(p.hw * CPG);
#pragma unroll
        for (int k = 0; k < Q; ++k) {
            if (lane == k) {
                const float rstd = 1.f / sqrtf(m[k].m2 / group_n + p.eps);
                const float hi = (float)m[k].mean, lo = (float)(m[k].mean - (double)hi);
                gstat[k][0] = hi;
                gstat[k][1] = lo;
                gstat[k][2] = rstd;
            }
        }
        __syncthreads();  // statistics in LDS
        if (lane < Q) ex_leave(p.ex, ng0 + lane, before);
    }
}

// --------------------------------------------------------------------------
// Host side.

// Elements per workgroup chunk for a dtype / vectorisation choice.
int64_t chunk_elems(kf_dtype xt, bool vector) {
    const int vec = vector ? (xt == KF_FLOAT32 ? 4 : 8) : 1;
    return (int64_t)kNT * (kFloatsPerThread / vec) * vec;
}

// 16-byte vectors: NCHW needs each channel's span to be whole vectors;
// channels last needs each group's channel run to be whole vectors and the
// channels of a thread to stay fixed across its slots (cpg divides
// 256 * VEC).  Both need 16-byte aligned bases.
bool vector_ok(const GroupNormArgs& a) {
    const int vec = a.xt == KF_FLOAT32 ? 4 : 8;
    if ((uintptr_t)a.x % 16 || (uintptr_t)a.y % 16) return false;
    const int64_t cpg = a.c / a.groups;
    if (a.nhwc) return cpg % vec == 0 && ((int64_t)kNT * vec) % cpg == 0;
    return a.spatial % vec == 0;
}

struct Layout {
    int64_t groups_total, parts;
    ExchangeLayout ex;
};

Layout layout(int64_t n, int64_t c, int64_t spatial, int64_t groups, kf_dtype xt, bool vector) {
    Layout l;
    l.groups_total = n * groups;
    const int64_t ge = (c / groups) * spatial;
    l.parts = (ge + chunk_elems(xt, vector) - 1) / chunk_elems(xt, vector);
    if (l.parts < 1) l.parts = 1;
    l.ex = exchange_layout(l.groups_total, l.parts);
    return l;
}

// KF355_GN_MODE selects the multi-chunk path: unset or "auto" (gn_pipe where
// it applies, else fused when resident, else two kernels), "fused" (as auto
// without gn_pipe), "coop" (fused only under a cooperative launch),
// "two_pass" (always two kernels).  Read once per process.
constexpr int kModeAuto = 0, kModeCoop = 1, kModeTwoPass = 2, kModeFused = 3;
int gn_mode() {
    static const int mode = [] {
        const char* e = std::getenv("KF355_GN_MODE");
        if (!e) return kModeAuto;
        if (!std::strcmp(e, "coop")) return kModeCoop;
        if (!std::strcmp(e, "two_pass")) return kModeTwoPass;
        if (!std::strcmp(e, "fused")) return kModeFused;
        return kModeAuto;
    }();
    return mode;
}

// KF355_GN_PARTS (tests only): gn_pipe with exactly this many workgroups per
// group where a chunk size gives it, including 1 (0 or unset: the default
// plan).  Read once per process.
uint32_t gn_parts_override() {
    static const uint32_t parts = env_u32("KF355_GN_PARTS", 0u);
    return parts;
}

// KF355_GN_ROUNDS (tests only): the fewest rounds gn_pipe may use (1 or 2;
// unset: 1).  Read once per process.
uint32_t gn_min_rounds() {
    static const uint32_t rounds = env_u32("KF355_GN_ROUNDS", 1u);
    return rounds;
}

// How long (100 MHz ticks of s_memrealtime) the second half of a one-round
// gn_pipe grid with at least two workgroups per CU waits before issuing its
// loads: 0.75 us by default; KF355_GN_STAGGER_TICKS overrides it (0: no
// wait).  On the SD3.5 VAE block (512 workgroups on 256 CUs, graph replays,
// three runs each): no wait 8.31-8.35 us; 0.6, 0.75 and 0.9 us 7.91-7.97;
// 1.25 us 8.25, 1.5 us 8.40, 2 us 8.94.  Waiting for one probe load of its
// own chunk instead of a fixed time gave 8.05-8.28 (two chained probe loads
// 8.56), delaying the last 5/8 or 3/8 of the grid instead of the half 8.30
// and 8.06, and a wait growing with the group index 8.19 at best.  The same
// wait on gn_pipe_cl (whose strided tiles bound it) gained 1%, so it stays
// on gn_pipe.  Read once per process.
uint32_t gn_stagger_ticks() {
    static const uint32_t ticks = env_u32("KF355_GN_STAGGER_TICKS", 75u);
    return ticks;
}

// KF355_GN_SPLIT_RECOMPUTE=1 (tests only): gn_split's last arrival of each
// group recomputes every part from x as it does when a published part stays
// unseen, and counts a give-up.  Read once per process.
bool gn_split_recompute() {
    static const bool on = env_u32("KF355_GN_SPLIT_RECOMPUTE", 0u) != 0;
    return on;
}

// How long (100 MHz ticks of s_memrealtime) a fused workgroup waits for the
// rest of its group before recomputing the statistics itself: 100 us by
// default; KF355_GN_WAIT_TICKS overrides it (tests set 0 to force the
// recompute path).  Read once per process.
uint32_t gn_wait_ticks() {
    static const uint32_t ticks = env_u32("KF355_GN_WAIT_TICKS", 10000u);
    return ticks;
}

// The exchange of a launch with `parts` parts per group (the give-up count
// at offset 0 of the workspace on every path).
Exchange gn_exchange(const GroupNormArgs& a, int64_t parts, int stride = 1) {
    return exchange_view(a.workspace, exchange_layout(a.n * a.groups, parts, stride), parts, gn_wait_ticks(), stride);
}

template <class T, class A, bool VECTOR, bool NHWC>
kf_status run(const GroupNormArgs& a, hipStream_t s, const char** variant) {
    const Layout l = layout(a.n, a.c, a.spatial, a.groups, a.xt, VECTOR);
    GNParams p;
    p.x = a.x;
    p.y = a.y;
    p.w = a.weight;
    p.b = a.bias;
    p.ex = gn_exchange(a, l.parts);
    p.group_elems = (a.c / a.groups) * a.spatial;
    p.spatial = a.spatial;
    p.channels = a.c;
    p.cpg = (int32_t)(a.c / a.groups);
    p.groups = (int32_t)a.groups;
    p.xcd_map = (!NHWC && l.groups_total % 8 == 0) ? 1 : 0;
    p.eps = a.eps;

    const int64_t grid = l.groups_total * l.parts;
    if (grid > INT32_MAX) {
        set_error("group_norm: grid of %lld workgroups exceeds the launch limit", (long long)grid);
        return KF_ERR_UNSUPPORTED_LAYOUT;
    }

    // Path choice.  One chunk per group needs no exchange.  Otherwise the
    // fused kernel is used when the occupancy-derived capacity covers the
    // grid (so normally every workgroup is resident and the exchange
    // completes; when it is not, the waiting workgroups recompute the
    // statistics themselves), launched normally, or cooperatively under
    // KF355_GN_MODE=coop.  In-place calls and grids larger than the
    // capacity take the two-kernel path.
    const int mode = gn_mode();
    enum { FUSED_SINGLE, FUSED_PLAIN, FUSED_COOP, TWO_PASS } path = TWO_PASS;
    if (l.parts == 1 && mode != kModeTwoPass) {
        path = FUSED_SINGLE;
    } else if (mode != kModeTwoPass && a.x != a.y) {
        static ResidencyCache capacity_cache;
        int dev = -1;
        if (hipGetDevice(&dev) != hipSuccess) {
            set_error("group_norm: no current HIP device");
            return KF_ERR_HIP;
        }
        const void* kernel = reinterpret_cast<const void*>(gn_fused<T, A, VECTOR, NHWC>);
        if ((int64_t)resident_capacity(capacity_cache, dev, kernel, kNT) >= grid) {
            if (mode == kModeCoop && device_cooperative(dev)) path = FUSED_COOP;
            else if (mode != kModeCoop) path = FUSED_PLAIN;
        }
    }
    // Variant names: [layout][vector][path].
    static const char* names[2][2][4] = {
        {{"gn_fused_scalar_single", "gn_fused_scalar", "gn_fused_scalar_coop", "gn_two_pass_scalar"},
         {"gn_fused_vec_single", "gn_fused_vec", "gn_fused_vec_coop", "gn_two_pass_vec"}},
        {{"gn_nhwc_fused_scalar_single", "gn_nhwc_fused_scalar", "gn_nhwc_fused_scalar_coop",
          "gn_nhwc_two_pass_scalar"},
         {"gn_nhwc_fused_vec_single", "gn_nhwc_fused_vec", "gn_nhwc_fused_vec_coop", "gn_nhwc_two_pass_vec"}}};
    *variant = names[NHWC ? 1 : 0][VECTOR ? 1 : 0][path];
    hipError_t err;
    if (path == FUSED_SINGLE || path == FUSED_PLAIN) {
        hipLaunchKernelGGL((gn_fused<T, A, VECTOR, NHWC>), dim3((unsigned)grid), dim3(kNT), 0, s, p);
        err = hipGetLastError();
    } else if (path == FUSED_COOP) {
        void* args[] = {&p};
        err = hipLaunchCooperativeKernel(reinterpret_cast<const void*>(gn_fused<T, A, VECTOR, NHWC>),
                                         dim3((unsigned)grid), dim3(kNT), args, 0, s);
    } else {
        hipLaunchKernelGGL((gn_stats<T, VECTOR, NHWC>), dim3((unsigned)grid), dim3(kNT), 0, s, p);
        err = hipGetLastError();
        if (err == hipSuccess) {
            hipLaunchKernelGGL((gn_apply<T, A, VECTOR, NHWC>), dim3((unsigned)grid), dim3(kNT), 0, s, p);
            err = hipGetLastError();
        }
    }
    if (err != hipSuccess) {
        set_error("group_norm launch failed: %s", hipGetErrorString(err));
        return KF_ERR_HIP;
    }
    return KF_OK;
}

// gn_pipe for dense NCHW 16-bit tensors, not in place, on 16-byte aligned
// bases, whose spatial size is a multiple of 2048 (every slot row of a
// chunk lies inside one channel) and whose groups split into 2 to 64 chunks,
// a power of two (the gather's lane butterfly).  Chunks of 16384 elements
// (8 slots per thread), else 32768 (16); one round when the grid of
// (groups x parts) workgroups is resident, else two.  Returns false, having
// launched nothing, when the shape is outside this.
template <class T, class A, int NV, int R>
const void* pipe_kernel() {
    return reinterpret_cast<const void*>(gn_pipe<T, A, NV, R>);
}

template <class T, class A>
bool run_pipe(const GroupNormArgs& a, hipStream_t s, const char** variant, kf_status* status) {
    const int mode = gn_mode();
    if (mode == kModeTwoPass || mode == kModeFused || mode == kModeCoop) return false;
    if (a.nhwc || a.x == a.y || !vector_ok(a) || a.spatial % 2048 != 0) return false;
    const int64_t ge = (a.c / a.groups) * a.spatial;
    const int64_t gt = a.n * a.groups;
    const int64_t forced = gn_parts_override();
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return false;
    static ResidencyCache cap[4][2];
    static const int nvs[4] = {8, 16, 4, 2};
    static const void* kernels[4][2] = {{pipe_kernel<T, A, 8, 1>(), pipe_kernel<T, A, 8, 2>()},
                                        {pipe_kernel<T, A, 16, 1>(), pipe_kernel<T, A, 16, 2>()},
                                        {pipe_kernel<T, A, 4, 1>(), pipe_kernel<T, A, 4, 2>()},
                                        {pipe_kernel<T, A, 2, 1>(), pipe_kernel<T, A, 2, 2>()}};
    static const char* names[4][2] = {{"gn_pipe_nv8_r1", "gn_pipe_nv8_r2"},
                                      {"gn_pipe_nv16_r1", "gn_pipe_nv16_r2"},
                                      {"gn_pipe_nv4_r1", "gn_pipe_nv4_r2"},
                                      {"gn_pipe_nv2_r1", "gn_pipe_nv2_r2"}};
    // The default plan tries 16384- then 32768-element chunks; an override
    // may also use 8192 and 4096.
    const int tries = forced ? 4 : 2;
    for (int k = 0; k < tries; ++k) {
        const int64_t ch = 2048 * (int64_t)nvs[k];
        if (ge % ch != 0) continue;
        const int64_t parts = ge / ch;
        if (forced ? parts != forced : parts < 2) continue;
        if (parts > 64 || (parts & (parts - 1)) != 0) continue;
        // The default chunks never need more exchange workspace than
        // kf_group_norm_workspace_bytes reports; a forced smaller chunk must
        // fit the caller's workspace, which must then not reach x or y.
        const size_t ws_need = exchange_layout(gt, parts).total;
        if (ws_need > a.workspace_bytes) continue;
        if (forced) {
            const uintptr_t w0 = (uintptr_t)a.workspace, w1 = w0 + ws_need;
            const uintptr_t bytes = (uintptr_t)(a.n * a.c * a.spatial * 2);
            const uintptr_t x0 = (uintptr_t)a.x, y0 = (uintptr_t)a.y;
            if ((w0 < x0 + bytes && x0 < w1) || (w0 < y0 + bytes && y0 < w1)) continue;
        }
        for (int r = gn_min_rounds() >= 2 ? 1 : 0; r < 2; ++r) {
            const int64_t rounds = r + 1;
            const int64_t per_round = (gt + rounds - 1) / rounds;
            const int64_t grid = per_round * parts;
            if (grid > INT32_MAX || (int64_t)resident_capacity(cap[k][r], dev, kernels[k][r], kPipeNT) < grid)
                continue;
            PipeParams p;
            p.x = a.x;
            p.y = a.y;
            p.w = a.weight;
            p.b = a.bias;
            p.ex = gn_exchange(a, parts);
            p.group_elems = ge;
            p.spatial = a.spatial;
            p.cpg = (int32_t)(a.c / a.groups);
            p.groups = (int32_t)a.groups;
            p.groups_total = (int32_t)gt;
            p.per_round = (int32_t)per_round;
            const bool stagger = rounds == 1 && grid >= 2 * (int64_t)device_multiprocessors(dev) && gn_stagger_ticks() > 0;
            p.stagger_from = stagger ? (int32_t)(grid / 2) : INT32_MAX;
            p.stagger_ticks = gn_stagger_ticks();
            p.force_recompute = 0;
            p.eps = a.eps;
            const dim3 g((unsigned)grid), b(kPipeNT);
            switch (k * 2 + r) {
                case 0: hipLaunchKernelGGL((gn_pipe<T, A, 8, 1>), g, b, 0, s, p); break;
                case 1: hipLaunchKernelGGL((gn_pipe<T, A, 8, 2>), g, b, 0, s, p); break;
                case 2: hipLaunchKernelGGL((gn_pipe<T, A, 16, 1>), g, b, 0, s, p); break;
                case 3: hipLaunchKernelGGL((gn_pipe<T, A, 16, 2>), g, b, 0, s, p); break;
                case 4: hipLaunchKernelGGL((gn_pipe<T, A, 4, 1>), g, b, 0, s, p); break;
                case 5: hipLaunchKernelGGL((gn_pipe<T, A, 4, 2>), g, b, 0, s, p); break;
                case 6: hipLaunchKernelGGL((gn_pipe<T, A, 2, 1>), g, b, 0, s, p); break;
                default: hipLaunchKernelGGL((gn_pipe<T, A, 2, 2>), g, b, 0, s, p); break;
            }
            const hipError_t err = hipGetLastError();
            *variant = names[k][r];
            if (err != hipSuccess) {
                set_error("group_norm launch failed: %s", hipGetErrorString(err));
                *status = KF_ERR_HIP;
            } else {
                *status = KF_OK;
            }
            return true;
        }
    }
    return false;
}

// Parts per group of gn_pipe_cl for a channels-last shape (the tile columns
// split each sample's pixels into hw / 256 parts), or 0 where it does not
// apply by shape: c a multiple of 64, cpg in {8, 16, 32, 64}, hw a multiple
// of 256 giving 2 to 64 parts, a power of two (the gather's butterfly).
int64_t cl_parts(int64_t c, int64_t spatial, int64_t groups) {
    const int64_t cpg = c / groups;
    if (c % 64 != 0 || (cpg != 8 && cpg != 16 && cpg != 32 && cpg != 64)) return 0;
    if (spatial % kClPixels != 0) return 0;
    const int64_t parts = spatial / kClPixels;
    if (parts < 2 || parts > 64 || (parts & (parts - 1)) != 0) return 0;
    return parts;
}

// gn_pipe_cl for dense channels-last 16-bit tensors, not in place, on
// 16-byte aligned bases, whose shape cl_parts admits and whose grid of
// (n * c / 64) * parts workgroups is resident.  Returns false, having
// launched nothing, otherwise.
template <class T, class A, int CPG>
const void* cl_kernel() {
    return reinterpret_cast<const void*>(gn_pipe_cl<T, A, CPG>);
}

template <class T, class A>
bool run_pipe_cl(const GroupNormArgs& a, hipStream_t s, const char** variant, kf_status* status) {
    const int mode = gn_mode();
    if (mode == kModeTwoPass || mode == kModeFused || mode == kModeCoop) return false;
    if (!a.nhwc || a.x == a.y || !vector_ok(a) || gn_parts_override()) return false;
    const int64_t parts = cl_parts(a.c, a.spatial, a.groups);
    if (!parts) return false;
    const int64_t gt = a.n * a.groups;
    if (exchange_layout(gt, parts, kClSlotStride).total > a.workspace_bytes) return false;
    const int64_t tiles = a.n * (a.c / 64);
    const int64_t grid = tiles * parts;
    if (grid > INT32_MAX || a.n * a.spatial > INT32_MAX) return false;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return false;
    const int cpg = (int)(a.c / a.groups);
    const int ci = cpg == 8 ? 0 : cpg == 16 ? 1 : cpg == 32 ? 2 : 3;
    static ResidencyCache cap[4];
    static const void* kernels[4] = {cl_kernel<T, A, 8>(), cl_kernel<T, A, 16>(), cl_kernel<T, A, 32>(),
                                     cl_kernel<T, A, 64>()};
    static const char* names[4] = {"gn_pipe_cl_cpg8", "gn_pipe_cl_cpg16", "gn_pipe_cl_cpg32", "gn_pipe_cl_cpg64"};
    if ((int64_t)resident_capacity(cap[ci], dev, kernels[ci], kPipeNT) < grid) return false;
    PipeClParams p;
    p.x = a.x;
    p.y = a.y;
    p.w = a.weight;
    p.b = a.bias;
    p.ex = gn_exchange(a, parts, kClSlotStride);
    p.hw = a.spatial;
    p.c = (int32_t)a.c;
    p.groups = (int32_t)a.groups;
    p.tiles_total = (int32_t)tiles;
    p.eps = a.eps;
    const dim3 g((unsigned)grid), b(kPipeNT);
    switch (ci) {
        case 0: hipLaunchKernelGGL((gn_pipe_cl<T, A, 8>), g, b, 0, s, p); break;
        case 1: hipLaunchKernelGGL((gn_pipe_cl<T, A, 16>), g, b, 0, s, p); break;
        case 2: hipLaunchKernelGGL((gn_pipe_cl<T, A, 32>), g, b, 0, s, p); break;
        default: hipLaunchKernelGGL((gn_pipe_cl<T, A, 64>), g, b, 0, s, p); break;
    }
    const hipError_t err = hipGetLastError();
    *variant = names[ci];
    if (err != hipSuccess) {
        set_error("group_norm launch failed: %s", hipGetErrorString(err));
        *status = KF_ERR_HIP;
    } else {
        *status = KF_OK;
    }
    return true;
}

// gn_split for dense NCHW 16-bit tensors that gn_pipe cannot take: 16384-
// element chunks (a multiple of 2048 spatial, so every slot row lies in one
// channel), a power-of-two number of 2 to 4096 parts per group, any grid
// size (nothing waits on another workgroup's progress), in place or not.
template <class T, class A>
bool run_split(const GroupNormArgs& a, hipStream_t s, const char** variant, kf_status* status) {
    constexpr int NV = 8;
    constexpr int64_t CH = (int64_t)kPipeDataWaves * kWave * NV * 8;
    const int mode = gn_mode();
    if (mode == kModeTwoPass || mode == kModeFused || mode == kModeCoop || gn_parts_override() != 0) return false;
    if (a.nhwc || !vector_ok(a) || a.spatial % 2048 != 0) return false;
    if (a.x != a.y) {  // exact aliasing is fine (each chunk is read before it is written); no partial overlap
        const uintptr_t bytes = (uintptr_t)(a.n * a.c * a.spatial * 2);
        const uintptr_t x0 = (uintptr_t)a.x, y0 = (uintptr_t)a.y;
        if (x0 < y0 + bytes && y0 < x0 + bytes) return false;
    }
    const int64_t ge = (a.c / a.groups) * a.spatial;
    if (ge % CH != 0) return false;
    const int64_t parts = ge / CH;
    if (parts < 2 || parts > 4096 || (parts & (parts - 1)) != 0) return false;
    const int64_t gt = a.n * a.groups;
    const int64_t grid = gt * parts;
    if (grid > INT32_MAX) return false;
    if (exchange_layout(gt, parts).total > a.workspace_bytes) return false;
    PipeParams p;
    p.x = a.x;
    p.y = a.y;
    p.w = a.weight;
    p.b = a.bias;
    p.ex = gn_exchange(a, parts);
    p.group_elems = ge;
    p.spatial = a.spatial;
    p.cpg = (int32_t)(a.c / a.groups);
    p.groups = (int32_t)a.groups;
    p.groups_total = (int32_t)gt;
    p.per_round = (int32_t)gt;
    p.stagger_from = INT32_MAX;
    p.stagger_ticks = 0;
    p.force_recompute = gn_split_recompute() ? 1 : 0;
    p.eps = a.eps;
    const dim3 g((unsigned)grid), b(kPipeDataWaves * kWave);
    hipLaunchKernelGGL((gn_split_stats<T, NV>), g, b, 0, s, p);
    hipError_t err = hipGetLastError();
    if (err == hipSuccess) {
        hipLaunchKernelGGL((gn_split_apply<T, A, NV>), g, b, 0, s, p);
        err = hipGetLastError();
    }
    *variant = "gn_split_nv8";
    if (err != hipSuccess) {
        set_error("group_norm launch failed: %s", hipGetErrorString(err));
        *status = KF_ERR_HIP;
    } else {
        *status = KF_OK;
    }
    return true;
}

template <class T, class A>
kf_status run_layout(const GroupNormArgs& a, hipStream_t s, const char** variant) {
    if constexpr (!std::is_same_v<T, F32>) {
        kf_status st;
        if (run_pipe<T, A>(a, s, variant, &st)) return st;
        if (run_pipe_cl<T, A>(a, s, variant, &st)) return st;
        if (run_split<T, A>(a, s, variant, &st)) return st;
    }
    const bool vec = vector_ok(a);
    if (a.nhwc) return vec ? run<T, A, true, true>(a, s, variant) : run<T, A, false, true>(a, s, variant);
    return vec ? run<T, A, true, false>(a, s, variant) : run<T, A, false, false>(a, s, variant);
}

// The exchange workspace of kf_group_norm_static: one array per GPU, in
// device memory from the moment this code object is loaded on that GPU until
// the process ends, zero-initialised at load (static storage) and returned
// to zero by every completed call, like a caller's workspace.  Host code must
// never pass `scratch` itself to a kernel or a copy (on the host the name
// stands for a host-side shadow, not a device address): it uses the device
// address hipGetSymbolAddress reports for the current device.
static __device__ __align__(256) unsigned char scratch[KF_GROUP_NORM_STATIC_SCRATCH_BYTES];

}  // namespace

kf_status group_norm_static_scratch(void** ptr) {
    constexpr int kDevices = 64;
    static std::atomic<void*> addr[kDevices];
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kDevices) {
        set_error("group_norm_static: no usable current HIP device (%d)", dev);
        return KF_ERR_HIP;
    }
    void* p = addr[dev].load(std::memory_order_acquire);
    if (!p) {
        // With `dev` current: each GPU holds its own copy at its own address.
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) {
            set_error("group_norm_static: hipGetSymbolAddress of the scratch array failed on device %d: %s", dev,
                      hipGetErrorString(e));
            return KF_ERR_HIP;
        }
        addr[dev].store(p, std::memory_order_release);
    }
    *ptr = p;
    return KF_OK;
}

size_t group_norm_workspace_bytes_for(int64_t n, int64_t c, int64_t spatial, int64_t groups, kf_dtype xt,
                                      bool nhwc) {
    // The scalar layout has the smallest chunk gn_fused uses, hence the most
    // parts, and the chunks of gn_pipe (default) and gn_split are no smaller;
    // gn_pipe_cl (channels-last 16-bit tensors) splits a group into more
    // parts, each slot on a line of its own.
    const size_t fused = layout(n, c, spatial, groups, xt, false).ex.total;
    const int64_t cl = !nhwc || xt == KF_FLOAT32 ? 0 : cl_parts(c, spatial, groups);
    const size_t tiles = cl ? exchange_layout(n * groups, cl, kClSlotStride).total : 0;
    return fused > tiles ? fused : tiles;
}

size_t group_norm_workspace_bytes(int64_t n, int64_t c, int64_t spatial, int64_t groups, kf_dtype xt) {
    // The query does not see the layout, so it covers both: one workspace
    // serves every path.
    return group_norm_workspace_bytes_for(n, c, spatial, groups, xt, true);
}

kf_status group_norm_launch(const GroupNormArgs& a, hipStream_t s, const char** variant) {
    const bool f32_affine = (a.at == KF_FLOAT32);
    switch (a.xt) {
        case KF_FLOAT32:
            return run_layout<F32, F32>(a, s, variant);
        case KF_BFLOAT16:
            return f32_affine ? run_layout<BF16, F32>(a, s, variant) : run_layout<BF16, BF16>(a, s, variant);
        case KF_FLOAT16:
            return f32_affine ? run_layout<F16, F32>(a, s, variant) : run_layout<F16, F16>(a, s, variant);
    }
    set_error("group_norm: unsupported dtype");
    return KF_ERR_BAD_DTYPE;
}

}  // namespace kf
