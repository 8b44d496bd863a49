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
//   gn_fused  (one launch, one HBM read + one write)  Each workgroup keeps its
//             chunk in registers, computes its (count, mean, M2) moments,
//             publishes them as one 64-bit word in its workspace slot, polls
//             the slots of its group until all `parts` are published, merges
//             them in part order (so the result does not depend on arrival
//             order), and normalises straight from registers.  Needs every
//             workgroup of the grid resident at once.
//   gn_stats + gn_apply  (two launches)  The same chunking without the wait:
//             the first kernel publishes the partials, the second merges them
//             and re-reads x.  Used when the grid cannot be co-resident.
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

// KF355_GN_MODE selects the multi-chunk path: unset or "auto" (fused when
// resident, else two kernels), "coop" (fused only under a cooperative
// launch), "two_pass" (always two kernels).  Read once per process.
constexpr int kModeAuto = 0, kModeCoop = 1, kModeTwoPass = 2;
int gn_mode() {
    static const int mode = [] {
        const char* e = std::getenv("KF355_GN_MODE");
        if (!e) return kModeAuto;
        if (!std::strcmp(e, "coop")) return kModeCoop;
        if (!std::strcmp(e, "two_pass")) return kModeTwoPass;
        return kModeAuto;
    }();
    return mode;
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
Exchange gn_exchange(const GroupNormArgs& a, int64_t parts) {
    return exchange_view(a.workspace, exchange_layout(a.n * a.groups, parts), parts, gn_wait_ticks());
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

template <class T, class A>
kf_status run_layout(const GroupNormArgs& a, hipStream_t s, const char** variant) {
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

size_t group_norm_workspace_bytes(int64_t n, int64_t c, int64_t spatial, int64_t groups, kf_dtype xt) {
    // The scalar layout has the smaller chunk, hence more parts: size for it
    // so one workspace serves either path.
    return layout(n, c, spatial, groups, xt, false).ex.total;
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
