// Memory-model primitives of the producer -> consumer handoff, shared by the
// all-reduce kernels and the litmus that checks them. gfx950 (MI355X) only.
//
// The 8 XCDs have separate L2s, so agent scope means "coherent across XCDs"
// (LLVM AMDGPU memory model for GFX942/950). A handoff publishes a slot's
// payload, then its stamps; the reader polls the stamps, then loads the
// payload. Partners on one XCD meet in that XCD's L2; partners on different
// XCDs need an agent-scope release before the stamps and an agent-scope
// acquire before the payload loads.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sifar {

struct alignas(16) V16 {
    uint32_t w[4];
};

__device__ __forceinline__ V16 ld16(const uint16_t *p) {
    return *reinterpret_cast<const V16 *>(p);
}

// `p`, the same in every lane of the wave, as a value the compiler knows to be
// wave-uniform (a scalar register pair), as a buffer descriptor needs.
// readfirstlane yields an int, so each half is taken as uint32_t: a low word
// with bit 31 set must not be sign-extended into the high word.
__device__ __forceinline__ const void *uniform_ptr(const void *p) {
    const uint64_t v = reinterpret_cast<uint64_t>(p);
    const uint32_t lo =
        static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v)));
    const uint32_t hi =
        static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v >> 32)));
    return reinterpret_cast<const void *>((static_cast<uint64_t>(hi) << 32) | lo);
}

// Buffer descriptor word 3 on gfx9-family GPUs: 32-bit data format, no
// swizzle, no thread-id addressing.
constexpr int32_t kBufferWord3 = 0x00020000;
// Cache policy of a buffer load: SC1 set, SC0 clear = agent scope.
constexpr int32_t kCachePolicyAgent = 16;

// Buffer descriptor of `base` (the same in every lane of the wave).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void *base) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(uniform_ptr(base)), 0, 0x7fffffff,
                                             kBufferWord3);
}

typedef int V4i __attribute__((ext_vector_type(4)));

// 16 bytes at byte offset `off` (per lane, below 2^31) from `base` (the same
// in every lane of the wave) through a buffer descriptor: the address lives in
// scalar registers and the only vector register the access reads is `off`.
// POLICY 0 caches normally; kCachePolicyAgent bypasses this CU's L1 (the
// caching of an agent-scope atomic load, in one 16-byte load instead of two
// 8-byte ones) and is served by the XCD's L2 or memory.
template <int POLICY>
__device__ __forceinline__ V16 ld16_buffer(const void *base, uint32_t off) {
    const V4i x = __builtin_amdgcn_raw_buffer_load_b128(buffer_rsrc(base), static_cast<int>(off),
                                                        0, POLICY);
    V16 v;
    v.w[0] = static_cast<uint32_t>(x[0]);
    v.w[1] = static_cast<uint32_t>(x[1]);
    v.w[2] = static_cast<uint32_t>(x[2]);
    v.w[3] = static_cast<uint32_t>(x[3]);
    return v;
}

__device__ __forceinline__ V16 ld16_agent(const void *base, uint32_t off) {
    return ld16_buffer<kCachePolicyAgent>(base, off);
}

// 16 bytes at byte offset off + soff through the descriptor rs, made once
// for several loads (per load only the scalar offset soff changes), with
// ld16_agent's caching: past this CU's L1.
__device__ __forceinline__ V16 ld16_agent_at(__amdgpu_buffer_rsrc_t rs, uint32_t off,
                                             uint32_t soff) {
    const V4i x = __builtin_amdgcn_raw_buffer_load_b128(rs, static_cast<int>(off),
                                                        static_cast<int>(soff), kCachePolicyAgent);
    V16 v;
    v.w[0] = static_cast<uint32_t>(x[0]);
    v.w[1] = static_cast<uint32_t>(x[1]);
    v.w[2] = static_cast<uint32_t>(x[2]);
    v.w[3] = static_cast<uint32_t>(x[3]);
    return v;
}

// 16 bytes to byte offset off + soff through the descriptor rs (normal
// caching), made once for several stores.
__device__ __forceinline__ void st16_at(__amdgpu_buffer_rsrc_t rs, uint32_t off, uint32_t soff,
                                        const V16 &v) {
    const V4i x = {static_cast<int>(v.w[0]), static_cast<int>(v.w[1]), static_cast<int>(v.w[2]),
                   static_cast<int>(v.w[3])};
    __builtin_amdgcn_raw_buffer_store_b128(x, rs, static_cast<int>(off), static_cast<int>(soff), 0);
}

// The store counterpart of ld16_buffer (normal caching).
__device__ __forceinline__ void st16_buffer(void *base, uint32_t off, const V16 &v) {
    const V4i x = {static_cast<int>(v.w[0]), static_cast<int>(v.w[1]), static_cast<int>(v.w[2]),
                   static_cast<int>(v.w[3])};
    __builtin_amdgcn_raw_buffer_store_b128(x, buffer_rsrc(base), static_cast<int>(off), 0, 0);
}

__device__ __forceinline__ void st16(uint16_t *p, const V16 &v) {
    *reinterpret_cast<V16 *>(p) = v;
}

// A 16-byte store of data no wave of the launch reads again (an all-reduce
// output): non-temporal, so that a large output stream does not push the slots
// and sources that every epoch re-reads out of the caches.
__device__ __forceinline__ void st16_stream(uint16_t *p, const V16 &v) {
    const V4i x = {static_cast<int>(v.w[0]), static_cast<int>(v.w[1]), static_cast<int>(v.w[2]),
                   static_cast<int>(v.w[3])};
    __builtin_nontemporal_store(x, reinterpret_cast<V4i *>(p));
}

__device__ __forceinline__ uint32_t ld_relaxed(const uint32_t *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ uint32_t ld_acquire(const uint32_t *p) {
    return __hip_atomic_load(p, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void st_relaxed(uint32_t *p, uint32_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// A flag for a partner wave on this XCD: a plain store lands in the XCD's L2,
// where the partner's agent-scope loads read it; an agent-scope store is
// written past the L2 and becomes visible to a poller later.
__device__ __forceinline__ void st_flag(uint32_t *p, uint32_t v, bool local) {
    if (local)
        __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    else
        __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void st_release(uint32_t *p, uint32_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}

// Makes every load that fed `v` complete before any later instruction issues:
// the value is consumed by an (empty) compiler barrier, so the compiler must
// wait for it there.
__device__ __forceinline__ void complete(const V16 &v) {
    asm volatile("" ::"v"(v.w[0]), "v"(v.w[1]), "v"(v.w[2]), "v"(v.w[3]) : "memory");
}

constexpr uint32_t kPlaceSpins = 1u << 14;  // polls for a partner wave's placement tag

// Placement of a persistent step's waves. Workgroups are dealt to the 8 XCDs
// round robin, so a chunk's consumer and producer share an XCD when the
// plane offset is a multiple of 8 -- but the kernel reads where it runs
// (XCC_ID) instead of assuming it. At step start every wave publishes
// ((base + 1) << 32) | 0x100 | XCD for its chunk and plane; a wave then reads
// its partner's tag (bounded wait; a missing tag counts as another XCD).

__device__ __forceinline__ uint32_t xcc_id() {
    uint32_t v;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID, 0, 4)" : "=s"(v));
    return v;
}

__device__ __forceinline__ uint64_t place_tag(uint32_t base, uint32_t xcc) {
    return (static_cast<uint64_t>(base + 1u) << 32) | 0x100u | xcc;
}

__device__ __forceinline__ void publish_place(uint64_t *place, uint32_t base, int lane) {
    if (lane == 0)
        __hip_atomic_store(place, place_tag(base, xcc_id()), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
}

// Wave-uniform: does the partner wave whose tag is *place run on this XCD?
__device__ __forceinline__ bool partner_is_local(const uint64_t *place, uint32_t base, int lane) {
    uint32_t local = 0;
    if (lane == 0) {
        const uint64_t want = place_tag(base, xcc_id());
        uint64_t t = 0;
        for (uint32_t spins = 0; spins < kPlaceSpins; ++spins) {
            t = __hip_atomic_load(place, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if ((t >> 32) == (want >> 32)) break;
            __builtin_amdgcn_s_sleep(1);
        }
        local = t == want ? 1u : 0u;
    }
    return __builtin_amdgcn_readfirstlane(local) != 0;
}

// Per lane: does the wave whose tag is *place run on this XCD? (bounded wait)
__device__ __forceinline__ bool tag_is_local(const uint64_t *place, uint32_t base) {
    const uint64_t want = place_tag(base, xcc_id());
    uint64_t t = 0;
    for (uint32_t spins = 0; spins < kPlaceSpins; ++spins) {
        t = __hip_atomic_load(place, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if ((t >> 32) == (want >> 32)) break;
        __builtin_amdgcn_s_sleep(1);
    }
    return t == want;
}

// s_waitcnt immediate (gfx9 family: vmcnt in bits 3:0 and 15:14, expcnt 6:4,
// lgkmcnt 11:8) with the export and LDS/scalar counts at their maxima and the
// vector-memory count 0; OR in n < 16 to wait until at most n vector memory
// operations of the wave are outstanding.
constexpr int kWaitVm = 0x0F70;

// Publication of a producer's slot stores before its stamps. To a consumer on
// another XCD: an agent-scope release fence, which writes back this XCD's L2.
// To a consumer on this XCD: waiting until the stores have reached the L2 is
// enough, because the L2 is the point of coherence of all CUs of one XCD and
// the consumer's agent-scope loads bypass its CU's L1 (the threadgroup-split
// workgroup scope of the LLVM AMDGPU memory model rests on the same fact: its
// release waits for the stores, its acquire bypasses or invalidates L1).
__device__ __forceinline__ void publish_slot(bool local) {
    if (local) {
        __builtin_amdgcn_s_waitcnt(0);
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
    } else {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    }
}

// The reader's side of publish_slot, after its stamps read as fresh: from a
// partner on another XCD, an agent-scope acquire fence (it invalidates this
// XCD's stale lines, so the payload loads cannot be served from them); from a
// partner on this XCD nothing beyond ordering the loads after the polls, since
// the payload is read with agent-scope loads that bypass L1.
__device__ __forceinline__ void acquire_slot(bool local) {
    if (local)
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
    else
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
}

}  // namespace sifar
