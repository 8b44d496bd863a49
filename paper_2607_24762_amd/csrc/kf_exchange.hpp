// kf_exchange.hpp -- cross-workgroup exchange of one 64-bit partial result
// per workgroup, for kernels that split one reduction unit (a GroupNorm
// group, a long softmax row) over `parts` workgroups.  Every workgroup of a
// unit publishes its partial, gathers all `parts` partials of the unit, and
// merges them in part order, so the merged value does not depend on arrival
// order and every workgroup of the unit computes it bit for bit the same.
//
// Protocol.  A published word is never 0 (the value of an empty slot): the
// caller's encoding sets a flag bit.  Writing data and flag in one
// single-copy-atomic 64-bit store means a reader that sees a non-zero word
// sees the data, so no fences and no cache write-back / invalidation are
// needed; polls are relaxed agent-scope loads.  The last workgroup of a unit
// to depart (a per-unit counter) clears the unit's slots and the counter, so
// every launch leaves its slots and counters as it found them: all zero.
// Waits are bounded by the 100 MHz real-time clock; a workgroup that gives up
// must recompute the missing partials itself (the kernels do,
// bit-identically) and adds one to the give-up count.  That count is the
// first word of a 256-byte status block at offset 0 of every workspace,
// whatever the shape, so a count left by one call can never be taken for a
// published partial or a departure count by a later call of another shape
// sharing the workspace; it is informational and only the caller resets it.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace kf {

constexpr size_t kCounterStride = 256;  // bytes between two units' counters

struct Exchange {
    uint64_t* slot;       // [units * parts] published partials (stride words apart), 0 = empty
    unsigned* depart;     // one counter per unit, kCounterStride bytes apart
    unsigned* give_ups;   // workgroups that stopped waiting (cumulative)
    int32_t parts;        // workgroups per unit
    int32_t stride;       // 64-bit words from one slot to the next (1: packed)
    uint32_t wait_ticks;  // give up waiting after this many 100 MHz ticks
};

// Slot q of `unit`.
__device__ __forceinline__ uint64_t* ex_slot(const Exchange& ex, int64_t unit, int q) {
    return ex.slot + (unit * ex.parts + q) * ex.stride;
}

__device__ __forceinline__ unsigned* ex_counter(const Exchange& ex, int64_t unit) {
    return reinterpret_cast<unsigned*>(reinterpret_cast<char*>(ex.depart) + unit * (int64_t)kCounterStride);
}

__device__ __forceinline__ void ex_publish(const Exchange& ex, int64_t unit, int part, uint64_t word) {
    __hip_atomic_store(ex_slot(ex, unit, part), word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Slot q of `unit`; with `wait`, polls until it is published or until
// wait_ticks have passed since t0 (a value of s_memrealtime), in which case
// it returns 0.
__device__ __forceinline__ uint64_t ex_poll(const Exchange& ex, int64_t unit, int q, uint64_t t0, bool wait) {
    uint64_t* at = ex_slot(ex, unit, q);
    uint64_t w = __hip_atomic_load(at, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (wait) {
        while (w == 0) {
            if (__builtin_amdgcn_s_memrealtime() - t0 > ex.wait_ticks) break;
            __builtin_amdgcn_s_sleep(1);
            w = __hip_atomic_load(at, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
    return w;
}

// Departure, in two steps, by one thread of every workgroup of `unit` once
// the workgroup has read all the unit's slots (its loads returned before the
// merge that precedes this).  ex_depart counts the workgroup out and returns
// how many had left before it; ex_leave, given that count, lets the last one
// empty the slots and the counter.  Callers put their own stores between the
// two, so the atomic's round trip overlaps them instead of ending the
// workgroup's life.
__device__ __forceinline__ unsigned ex_depart(const Exchange& ex, int64_t unit) {
    return __hip_atomic_fetch_add(ex_counter(ex, unit), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void ex_leave(const Exchange& ex, int64_t unit, unsigned departed_before) {
    if (departed_before == (unsigned)ex.parts - 1) {
        for (int q = 0; q < ex.parts; ++q)
            __hip_atomic_store(ex_slot(ex, unit, q), (uint64_t)0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(ex_counter(ex, unit), 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

__device__ __forceinline__ void ex_release(const Exchange& ex, int64_t unit) { ex_leave(ex, unit, ex_depart(ex, unit)); }

__device__ __forceinline__ void ex_count_give_up(const Exchange& ex) {
    __hip_atomic_fetch_add(ex.give_ups, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ---------------------------------------------------------------------------
// Host side: workspace layout.  The 256-byte status block first (its first
// 32-bit word the give-up count; the rest unused), then the slots (`stride`
// words apart: 16 gives every slot a 128-byte line of its own), then one
// 256-byte line per unit for its counter (so different units never share a
// line).
constexpr size_t kStatusBytes = 256;

struct ExchangeLayout {
    size_t slot_off, depart_off, total;
};

inline ExchangeLayout exchange_layout(int64_t units, int64_t parts, int stride = 1) {
    auto up = [](size_t v) { return (v + 255) & ~(size_t)255; };
    ExchangeLayout l;
    l.slot_off = kStatusBytes;
    l.depart_off = l.slot_off + up((size_t)(units * parts * stride) * sizeof(uint64_t));
    l.total = l.depart_off + (size_t)units * kCounterStride;
    return l;
}

inline Exchange exchange_view(void* workspace, const ExchangeLayout& l, int64_t parts, uint32_t wait_ticks,
                              int stride = 1) {
    char* ws = static_cast<char*>(workspace);
    Exchange ex;
    ex.slot = reinterpret_cast<uint64_t*>(ws + l.slot_off);
    ex.depart = reinterpret_cast<unsigned*>(ws + l.depart_off);
    ex.give_ups = reinterpret_cast<unsigned*>(ws);
    ex.parts = (int32_t)parts;
    ex.stride = stride;
    ex.wait_ticks = wait_ticks;
    return ex;
}

}  // namespace kf
