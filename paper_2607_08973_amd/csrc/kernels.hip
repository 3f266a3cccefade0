// gfx950 (MI355X) kernels of the emulated SiFAR one-shot all-reduce.
//
// Work decomposition: a "chunk" is 512 consecutive bf16 elements of one
// token's row, handled by one 64-lane wave with one 16-byte load per rank per
// lane. Every chunk carries its own N epoch stamps (the paper's per-threadblock
// validation buffer, Sec. 4.2), so chunks validate and retry independently and
// no wave waits for another during the reduction proper.
//
// Two ways to run a decode step:
//  - per-epoch launches (eager calls, step graphs): the producer of an epoch
//    always finishes in an earlier launch than the reduction of that epoch, so
//    the paper's speculative reduction (SPEC) is exact here;
//  - one persistent launch per step (chain_kernel): consumer and producer
//    waves run concurrently and synchronise through stamps and per-chunk
//    consumed/produced words; the consumer validates before it loads
//    (ORDERED), since speculative loads racing a live producer were measured
//    to accept stale data.
//
// Memory-model choices (LLVM AMDGPU memory model for GFX942/950; the 8 XCDs
// have separate L2s, so agent scope means "coherent across XCDs"; the handoff
// primitives live in coherence.h, which the handoff litmus also runs):
//  - stamps are read with agent-scope atomic loads;
//  - per-epoch SPEC issues the payload loads and the stamp loads together (the
//    paper's concurrent payload warps and validation warp); ORDERED acquires
//    the stamps before loading the payload; a retry starts with an acquire
//    fence so the reloads cannot be served from a stale cache line (the
//    paper's L1-bypassing re-read, Sec. 4.2);
//  - in the persistent chain each wave learns whether its partner shares its
//    XCD. Same-XCD pairs meet in that XCD's L2: plain flag stores, a wait for
//    the slot stores instead of a release fence, agent-scope (L1-bypassing)
//    loads. Cross-XCD pairs use agent-scope stores, a release fence before the
//    stamps and an acquire fence before the payload loads.
//
// Arithmetic: fp32 adds in ascending rank order (no reassociation, no FMA
// contraction), bf16 rounding by the native V_CVT_PK_BF16_F32 (round to nearest
// even, fp32 denormals enabled).
#include "coherence.h"
#include "sifar_kernels.h"

namespace sifar {
namespace {

__device__ __forceinline__ float lo_f32(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_f32(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Two fp32 values to two bf16 in one V_CVT_PK_BF16_F32 (round to nearest
// even); converting them one at a time costs four instructions per pair.
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
    typedef float f32x2 __attribute__((ext_vector_type(2)));
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    const f32x2 f = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2));
}

__device__ __forceinline__ uint32_t epoch_of(const EpochRef &e) { return e.base[0] + e.off; }

// First error wins; kind 0 means "no error".
__device__ void latch(uint32_t *err, uint32_t kind, uint32_t g, uint32_t c, uint32_t n) {
    uint32_t expected = 0;
    if (__hip_atomic_compare_exchange_strong(err, &expected, kind, __ATOMIC_RELAXED,
                                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
        st_relaxed(err + 1, g);
        st_relaxed(err + 2, c);
        st_relaxed(err + 3, n);
    }
}

constexpr uint32_t kErrRetryBudget = 1, kErrWaw = 2, kErrExchange = 3;

// A persistent step's waits read the error word only once they have lasted
// this many polls, and no wave reads it otherwise: a healthy epoch needs one
// or two polls, so the word is never read, while a wave whose wait outlasts
// the step's failure elsewhere still leaves within microseconds. The word is
// one address for the whole GPU: read by every consumer wave once per epoch
// (beside its first stamp poll) it bounded the step as the chunks grew.
// Measured on MI355X (llama8b decode, N = 8, H = 4096, us per all-reduce):
// reading it with every poll, 0.794 at T = 1..8 / 1.01 at 16 tokens / 2.15 at
// 64 tokens; only after 64 polls, 0.784 / 0.98 / 2.13 while consumers still
// read it once per epoch; not per epoch either, 0.760 / 0.80 / 1.12.
constexpr uint32_t kErrPollAfter = 64;

// Where the calling lane works: token t, chunk s of the row, chunk index c.
// Lanes past the end of the row load a clamped, in-bounds address (the row's
// last 8 elements) and do not store (lane_ok false) -- except where a store of
// the very bytes the owning lane stores keeps a loop branch-free; waves past
// the last chunk are inactive.
struct Chunk {
    int t, s, c;
    bool active, lane_ok;
    int elem;
    uint64_t row;
};

__device__ __forceinline__ Chunk chunk_at(const Geometry &geo, int t, int s, int lane) {
    Chunk k;
    k.t = t;
    k.active = s < geo.segs;
    k.s = k.active ? s : geo.segs - 1;
    k.c = t * geo.segs + k.s;
    const int raw = s * kChunk + lane * kVec;
    k.lane_ok = k.active && raw < geo.hidden;
    const int e = k.s * kChunk + lane * kVec;
    k.elem = e < geo.hidden ? e : geo.hidden - kVec;
    k.row = static_cast<uint64_t>(t) * geo.hidden + k.elem;
    return k;
}

__device__ __forceinline__ uint32_t log_word(uint32_t attempts, uint32_t first, uint32_t last) {
    return (attempts > 0xFFFFu ? 0xFFFFu : attempts) | ((first & 0xFFu) << 16) |
           ((last & 0xFFu) << 24);
}

// The injection table's word for epoch g (late | withheld << 8), 0 without a
// table.
__device__ __forceinline__ uint32_t inject_word(const uint16_t *inject, const DivU32 &div,
                                                uint32_t g) {
    return inject ? inject[mod_u32(g - 1u, div)] : 0u;
}

// Ranks an injection word makes late (not withheld).
__device__ __forceinline__ uint32_t late_ranks(uint32_t inj) { return inj & ~(inj >> 8) & 0xFFu; }

// ---------------------------------------------------------------------------
// Producer side: the emulated peers.

// Index of chunk k's first element in a row-major [tokens][hidden] array
// (wave-uniform), and the calling lane's byte offset from it.
__device__ __forceinline__ uint64_t chunk_first(const Geometry &geo, const Chunk &k) {
    return static_cast<uint64_t>(k.t) * geo.hidden + static_cast<uint64_t>(k.s) * kChunk;
}

__device__ __forceinline__ uint32_t lane_offset(const Geometry &geo, const Chunk &k) {
    return static_cast<uint32_t>(k.row - chunk_first(geo, k)) * 2u;
}

// Every rank's part of chunk k of epoch g (the peers' partial results), read
// through buffer descriptors: the per-lane address is the loop-invariant
// offset, so no vector register of an access in flight is ever rewritten.
template <int N>
__device__ __forceinline__ void load_sources(const ProduceArgs &a, const Chunk &k, uint32_t g,
                                             V16 (&v)[N]) {
    const uint32_t e = mod_u32(g - 1u, a.entries_div);
    const uint16_t *src = a.src + e * a.entry_stride + static_cast<int64_t>(chunk_first(a.geo, k));
    const uint32_t off = lane_offset(a.geo, k);
#pragma unroll
    for (int r = 0; r < N; ++r) v[r] = ld16_buffer<0>(src + r * a.rank_stride, off);
}

// The same through one descriptor, every rank's slot at a scalar offset from
// rank 0's (launch_chain checks that the offsets fit): one scalar instruction
// per store instead of three for a descriptor of its own, so the stores the
// publication waits for leave back to back.
template <int N>
__device__ __forceinline__ void store_slots_at(const ProduceArgs &a, const Chunk &k, uint32_t p,
                                               const V16 (&v)[N]) {
    const Geometry &geo = a.geo;
    const __amdgpu_buffer_rsrc_t rs =
        buffer_rsrc(a.slots + static_cast<uint64_t>(p) * geo.slot_elems + chunk_first(geo, k));
    const uint32_t off = lane_offset(geo, k);
    const uint32_t rank_bytes = static_cast<uint32_t>(geo.slot_elems) * 4u;
    if (k.lane_ok) {
#pragma unroll
        for (int r = 0; r < N; ++r) st16_at(rs, off, static_cast<uint32_t>(r) * rank_bytes, v[r]);
    }
}

// ... written into the slots of parity p.
template <int N>
__device__ __forceinline__ void store_slots(const ProduceArgs &a, const Chunk &k, uint32_t p,
                                            const V16 (&v)[N]) {
    const Geometry &geo = a.geo;
    uint16_t *dst = a.slots + static_cast<uint64_t>(p) * geo.slot_elems + chunk_first(geo, k);
    const uint32_t off = lane_offset(geo, k);
    if (k.lane_ok) {
#pragma unroll
        for (int r = 0; r < N; ++r) st16_buffer(dst + r * 2 * geo.slot_elems, off, v[r]);
    }
}

// Copy every rank's part of chunk k of epoch g into the slots of parity p
// (the producers that load and store in one go; plain global addressing
// measured faster for them than the buffer form above). Ranks in `staged`
// (wave-uniform) write into the stage instead: they are late, and their slot
// keeps its previous epoch until they catch up.
template <int N>
__device__ __forceinline__ void copy_chunk(const ProduceArgs &a, const Chunk &k, uint32_t g,
                                           uint32_t p, uint32_t staged = 0) {
    const Geometry &geo = a.geo;
    const uint32_t e = mod_u32(g - 1u, a.entries_div);
    const uint16_t *src = a.src + e * a.entry_stride + static_cast<int64_t>(k.row);
    const uint64_t at = static_cast<uint64_t>(p) * geo.slot_elems + k.row;
    V16 v[N];
#pragma unroll
    for (int r = 0; r < N; ++r) v[r] = ld16(src + r * a.rank_stride);
    if (k.lane_ok) {
#pragma unroll
        for (int r = 0; r < N; ++r) {
            uint16_t *dst = ((staged >> r) & 1u) ? a.stage : a.slots;
            st16(dst + at + r * 2 * geo.slot_elems, v[r]);
        }
    }
}

// Ranks whose stamp an injection word holds back (late | withheld).
__device__ __forceinline__ uint32_t held_back(uint32_t inj) { return (inj | (inj >> 8)) & 0xFFu; }

// Producer of one epoch in its own launch (eager calls, step graphs). With
// deterministic injection a late rank's payload goes to the stage and its
// stamp is not written: the rank has not caught up yet. The
// stamp stores are ordered after the payload stores of the wave
// (workgroup-scope release); device-wide visibility comes from the end of the
// launch, because the reduction of an epoch always runs in a later launch than
// its producer (eagerly, in a step graph, and in the fused plane, which writes
// the epoch after the one its launch reduces) -- as in the paper, whose flag
// follows the preceding kernel's completion (Sec. 4.2). An agent-scope release
// here would write back the XCD's whole L2 once per wave; measured on MI355X
// that costs ~0.1-0.2 us of XCD-serialised time per fence and caps a 38 MB
// all-reduce at 0.9 TB/s instead of 5.7 TB/s. Workgroups are numbered
// chunk-fastest then token, the order the reduction numbers its chunks, so with
// one wave per group the producer and the reduction of a chunk share an XCD.
template <int N>
__device__ __forceinline__ void produce_chunk(const ProduceArgs &a, int G) {
    const int lane = threadIdx.x & (kLanes - 1);
    const Geometry &geo = a.geo;
    // The epoch first: the source address depends on it, and a uniform load
    // ahead of anything that may write memory stays a scalar load.
    const uint32_t g = epoch_of(a.ep);
    // Every other argument the wave reads before its source loads, requested
    // in one batch: the compiler otherwise loads kernel arguments block by
    // block, one memory round trip at a time (measured: 4-5 of them in a row
    // before the sources were requested).
    asm volatile("" ::"s"(geo.hidden), "s"(geo.segs), "s"(geo.w_max), "s"(geo.slot_elems),
                 "s"(a.ep.base), "s"(a.ep.parity), "s"(a.slots), "s"(a.stamps),
                 "s"(a.consumed), "s"(a.produced), "s"(a.src), "s"(a.entry_stride),
                 "s"(a.rank_stride), "s"(a.entries_div.m), "s"(a.entries_div.sh1),
                 "s"(a.entries_div.sh2), "s"(a.entries_div.d), "s"(a.inject), "s"(a.stage),
                 "s"(a.ep.off));
    const Chunk k = chunk_at(geo, blockIdx.y, blockIdx.x * G + threadIdx.x / kLanes, lane);
    if (!k.active) return;
    const uint32_t p = a.ep.parity;
    const size_t pc = static_cast<size_t>(p) * geo.w_max + k.c;
    // Dual-buffer rule: the slot's previous epoch must have been consumed.
    const uint32_t prev = ld_relaxed(a.produced + pc);
    const uint32_t done = ld_relaxed(a.consumed + pc);
    const uint32_t inj = inject_word(a.inject, a.inject_div, g);
    const uint32_t held = held_back(inj);
    copy_chunk<N>(a, k, g, p, a.stage ? late_ranks(inj) : 0u);
    if (lane == 0 && prev != done) latch(a.err, kErrWaw, g, k.c, prev);
    // The stamps follow the payload within the wave; the reduction reads them
    // in a later launch, whose start makes them visible device-wide, so they
    // need not be written past the L2 (an agent-scope store would make the
    // launch wait for that before it can end).
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    uint32_t *stamp = a.stamps + pc * N;
    if (lane < N && !((held >> lane) & 1u)) st_flag(stamp + lane, g, true);
    if (lane == 0) st_flag(a.produced + pc, g, true);
}

template <int N>
__global__ __launch_bounds__(1024) void produce_kernel(ProduceArgs a) {
    produce_chunk<N>(a, static_cast<int>(blockDim.x) / kLanes);
}

// ---------------------------------------------------------------------------
// Consumer side.

template <int N>
__device__ __forceinline__ void load_payload(V16 (&v)[N], const uint16_t *slot0, uint64_t rank_step) {
#pragma unroll
    for (int r = 0; r < N; ++r) v[r] = ld16(slot0 + r * rank_step);
}

// Gather of a per-epoch launch: load chunk k of epoch g, validate its N
// stamps, retry while any is stale. The epoch's on-time payload was written by
// an earlier launch, so a stale stamp can only be an injected late one.
// INJECT_HOOK: deterministic injection, the late ranks catch up right after
// the first failed validation: their payload moves from the stage into the
// slot (which still held their previous epoch when it was first loaded),
// then, after a release, their stamps are written. The retry must therefore
// reload the payload to get the right sum. `st_first` / `st_last`: this
// lane's stamp (lanes < N) at the first and at the last validation.
// `base_v` is the launch's epoch base as loaded (g = base_v + the launch's
// offset); its first use waits until the payload and stamp loads are issued.
template <int N, int MODE, bool INJECT_HOOK>
__device__ __forceinline__ uint32_t gather(const ReduceArgs &a, const Chunk &k, uint32_t base_v,
                                           uint32_t p, int lane, V16 (&v)[N], uint32_t &attempts,
                                           uint32_t &first, uint32_t &last, uint32_t &st_first,
                                           uint32_t &st_last) {
    const Geometry &geo = a.geo;
    const uint16_t *slot0 = a.slots + static_cast<uint64_t>(p) * geo.slot_elems + k.row;
    const uint64_t rank_step = 2 * geo.slot_elems;  // slots are [rank][parity]
    uint32_t *stamp = a.stamps + (static_cast<size_t>(p) * geo.w_max + k.c) * N;
    // every lane loads a stamp (lanes >= N rank N - 1's, which the ballot
    // ignores): no branch holds the loads back behind the epoch's arrival
    const uint32_t *stamp_lane = stamp + (lane < N ? lane : N - 1);

    uint32_t st = 0;
    if (MODE == kOrdered) {
        st = ld_acquire(stamp_lane);
    } else {
        load_payload<N>(v, slot0, rank_step);
        if (MODE == kSpec) st = ld_relaxed(stamp_lane);
    }
    // nothing that needs the epoch may move ahead of these loads (the compiler
    // otherwise waits for the epoch's load before it issues them)
    __builtin_amdgcn_sched_barrier(0);
    // the arguments needed once the payload is in, requested in one batch
    // while it travels (the compiler would otherwise load them one round trip
    // at a time where each is first used)
    asm volatile("" ::"s"(a.consumed), "s"(a.log), "s"(a.stamp_log), "s"(a.log_div.m),
                 "s"(a.log_div.sh1), "s"(a.log_div.sh2), "s"(a.log_div.d),
                 "s"(a.forced_retries), "s"(a.out), "s"(a.max_attempts), "s"(a.inject));
    const uint32_t g = base_v + a.ep.off;
    st_first = st;

    attempts = 1;
    first = last = 0;
    if (MODE != kNone && k.active) {
        uint32_t m = static_cast<uint32_t>(__ballot(lane < N && st != g));
        first = last = m;
        bool fail = m != 0 || a.forced_retries >= 1;
        while (fail) {
            if (attempts >= a.max_attempts) {
                if (lane == 0) latch(a.err, kErrRetryBudget, g, k.c, attempts);
                break;
            }
            if (INJECT_HOOK && attempts == 1 && a.inject && m != 0) {
                const uint32_t late = late_ranks(inject_word(a.inject, a.inject_div, g));
                if (a.stage) {
                    const uint64_t at = static_cast<uint64_t>(p) * geo.slot_elems + k.row;
#pragma unroll
                    for (int r = 0; r < N; ++r) {
                        if ((late >> r) & 1u) {
                            const V16 x = ld16(a.stage + at + r * rank_step);
                            if (k.lane_ok) st16(a.slots + at + r * rank_step, x);
                        }
                    }
                }
                // the payload is published before the stamps, as a peer would
                __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
                if (lane < N && ((late >> lane) & 1u)) st_relaxed(stamp + lane, g);
            }
            // plain reloads need an acquire fence (an L2 invalidate) to see the
            // peers' data
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
            if (MODE == kOrdered) {
                st = ld_acquire(stamp_lane);
            } else {
                st = ld_relaxed(stamp_lane);
                load_payload<N>(v, slot0, rank_step);
            }
            ++attempts;
            m = static_cast<uint32_t>(__ballot(lane < N && st != g));
            last = m;
            fail = m != 0 || attempts <= a.forced_retries;
        }
    }
    st_last = st;
    if (MODE == kOrdered) load_payload<N>(v, slot0, rank_step);
    return g;
}

// Persistent-step gather of an active chunk: a producer may be writing right
// now, so only ORDERED is sound. `m` is the stale-rank mask of the first stamp
// poll and `st` this lane's stamp from it (issued and evaluated by the
// caller); polls repeat (relaxed agent-scope loads; lanes >= N read rank
// N - 1's, which the ballot ignores) until every stamp is fresh, then the
// payload is loaded -- after an acquire fence when the producer is on another
// XCD, directly when it shares this XCD (see publish_slot). On return `st`
// holds the stamp of the last poll; the result is true when the wait failed:
// the retry budget ran out (latched here), or an error latched elsewhere was
// found while waiting. With AT the payload loads share one descriptor, every
// rank at a scalar offset, and leave back to back (a lone wave pays an issue
// slot for every instruction: three scalar ones per descriptor kept the last
// load ~50 ns behind the first). Epilogue kernels keep a descriptor per load:
// their scalar registers are full, and the hoisted offsets spilled into 12
// more vector registers. Measured with the producer's stores done the same
// way (llama8b decode, us per all-reduce): 0.759 -> 0.721 at T = 1..8,
// 0.80 -> 0.75 at 16 tokens, 1.13 -> 1.08 at 64 tokens.
template <int N, bool AT>
__device__ __forceinline__ bool gather_chain(const ReduceArgs &a, const Chunk &k, uint32_t g,
                                             uint32_t p, int lane, uint32_t m, uint32_t &st,
                                             V16 (&v)[N], uint32_t &attempts, uint32_t &first,
                                             uint32_t &last, bool local) {
    const Geometry &geo = a.geo;
    // the chunk's first element in rank 0's slot (wave-uniform) and this
    // lane's byte offset from it
    const uint16_t *chunk0 =
        a.slots + static_cast<uint64_t>(p) * geo.slot_elems + chunk_first(geo, k);
    const uint32_t off = lane_offset(geo, k);
    const uint64_t rank_step = 2 * geo.slot_elems;  // slots are [rank][parity]
    const uint32_t *stamp = a.stamps + (static_cast<size_t>(p) * geo.w_max + k.c) * N +
                            (lane < N ? lane : N - 1);
    attempts = 1;
    first = last = m;
    bool fail = m != 0 || a.forced_retries >= 1;
    bool failed = false;
    while (fail) {
        if (attempts >= a.max_attempts) {
            if (lane == 0) latch(a.err, kErrRetryBudget, g, k.c, attempts);
            failed = true;
            break;
        }
        // one round trip per poll, back to back (a short sleep between polls
        // measured ~2 % slower); the error word joins it after kErrPollAfter
        const uint32_t e = attempts >= kErrPollAfter ? ld_relaxed(a.err) : 0u;
        st = ld_relaxed(stamp);
        ++attempts;
        m = static_cast<uint32_t>(__ballot(lane < N && st != g));
        last = m;
        if (m != 0 && e != 0) {  // the step is already failing: stop waiting
            failed = true;
            break;
        }
        fail = m != 0 || attempts <= a.forced_retries;
    }
    acquire_slot(local);
    if (AT) {
        const __amdgpu_buffer_rsrc_t rs = buffer_rsrc(chunk0);
        const uint32_t rank_bytes = static_cast<uint32_t>(rank_step) * 2u;
#pragma unroll
        for (int r = 0; r < N; ++r)
            v[r] = ld16_agent_at(rs, off, static_cast<uint32_t>(r) * rank_bytes);
    } else {
#pragma unroll
        for (int r = 0; r < N; ++r) v[r] = ld16_agent(chunk0 + r * rank_step, off);
    }
    return failed;
}

// Fixed-order fp32 sum: acc = x_0; acc += x_1; ... acc += x_{N-1}; then bf16.
template <int N>
__device__ __forceinline__ V16 sum_round(const V16 (&v)[N]) {
    float acc[kVec];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        acc[2 * k] = lo_f32(v[0].w[k]);
        acc[2 * k + 1] = hi_f32(v[0].w[k]);
    }
#pragma unroll
    for (int r = 1; r < N; ++r) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            acc[2 * k] = acc[2 * k] + lo_f32(v[r].w[k]);
            acc[2 * k + 1] = acc[2 * k + 1] + hi_f32(v[r].w[k]);
        }
    }
    V16 o;
#pragma unroll
    for (int k = 0; k < 4; ++k) o.w[k] = pack_bf16(acc[2 * k], acc[2 * k + 1]);
    return o;
}

__device__ __forceinline__ void write_log(const ReduceArgs &a, const Chunk &k, uint32_t g,
                                          uint32_t word) {
    a.log[static_cast<size_t>(mod_u32(g - 1u, a.log_div)) * a.geo.w_max + k.c] =
        word;
}

// Rank r's raw stamp at the chunk's first and last validation, beside the
// decision word, so that every logged mask can be recomputed from the stamps.
template <int N>
__device__ __forceinline__ void write_stamp_log(const ReduceArgs &a, const Chunk &k, uint32_t g,
                                                int r, uint32_t first, uint32_t last) {
    uint32_t *row = a.stamp_log +
                    (static_cast<size_t>(mod_u32(g - 1u, a.log_div)) *
                         a.geo.w_max + k.c) * (2 * N) + r;
    row[0] = first;
    row[N] = last;
}

// Residual-add + RMSNorm of one chunk after its all-reduce result o. The
// token's sum of squares is combined across the waves of the workgroup (LDS)
// and across the token's Q workgroups (epoch-tagged exchange words, double
// buffered by the epoch's parity). Every wave of the workgroup must call this.
__device__ __forceinline__ void residual_rmsnorm(const ReduceArgs &a, const Chunk &k, uint32_t g,
                                                 const V16 &o, const V16 &rv,
                                                 const V16 &wv, uint16_t *y, int lane, int wave,
                                                 int G, int q, bool xlocal = false) {
    const Geometry &geo = a.geo;
    // res' = bf16(a + res), with a = the bf16 all-reduce result.
    V16 nr;
    float x[kVec];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float a0 = lo_f32(o.w[i]), a1 = hi_f32(o.w[i]);
        nr.w[i] = pack_bf16(a0 + lo_f32(rv.w[i]), a1 + hi_f32(rv.w[i]));
        x[2 * i] = lo_f32(nr.w[i]);
        x[2 * i + 1] = hi_f32(nr.w[i]);
    }
    if (k.lane_ok) st16(a.residual + k.row, nr);

    float ss = 0.f;
    if (k.lane_ok) {
#pragma unroll
        for (int i = 0; i < kVec; ++i) ss = __builtin_fmaf(x[i], x[i], ss);
    }
    // Butterfly: every lane ends with the bit-identical wave total.
#pragma unroll
    for (int off = kLanes / 2; off >= 1; off >>= 1) ss = ss + __shfl_xor(ss, off);

    __shared__ float part[kMaxWavesPerGroup];
    __shared__ float total;
    if (lane == 0) part[wave] = ss;  // idle waves contribute 0
    __syncthreads();
    float grp = 0.f;
    for (int w = 0; w < G; ++w) grp = grp + part[w];

    const int Q = a.groups_per_token;
    if (Q > 1) {
        if (wave == 0) {
            uint64_t *ex = a.exch + static_cast<size_t>(g & 1u) * a.exch_parity_stride +
                           static_cast<size_t>(k.t) * Q;
            if (lane == 0) {
                const uint64_t word = (static_cast<uint64_t>(g) << 32) | __float_as_uint(grp);
                // all groups of the token on this XCD: the word meets them in its L2
                if (xlocal)
                    __hip_atomic_store(ex + q, word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
                else
                    __hip_atomic_store(ex + q, word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
            uint64_t mine = 0;
            uint32_t spins = 0;
            bool ready;
            do {
                if (lane < Q)
                    mine = __hip_atomic_load(ex + lane, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                ready = __ballot(lane < Q && static_cast<uint32_t>(mine >> 32) != g) == 0;
            } while (!ready && ++spins < a.spin_limit);
            if (!ready && lane == 0) latch(a.err, kErrExchange, g, k.c, spins);
            const float pv = __uint_as_float(static_cast<uint32_t>(mine));
            float tot = 0.f;
            for (int j = 0; j < Q; ++j) tot = tot + __shfl(pv, j);
            if (lane == 0) total = tot;
        }
        __syncthreads();
        grp = total;
    }

    const float inv = 1.0f / __builtin_sqrtf(grp / static_cast<float>(geo.hidden) + a.eps);
    V16 yo;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float w0 = lo_f32(wv.w[i]), w1 = hi_f32(wv.w[i]);
        yo.w[i] = pack_bf16((x[2 * i] * inv) * w0, (x[2 * i + 1] * inv) * w1);
    }
    if (k.lane_ok) st16(y + k.row, yo);
}

// ---------------------------------------------------------------------------
// Reduction of one epoch, one chunk per wave: speculative or ordered loads,
// per-rank stamp validation by ballot, bounded retry, fp32 sum in rank order,
// bf16 store, optional fused epilogue.
// FUSED: the grid has a second plane (blockIdx.z == 1) of producer workgroups
// that write the NEXT epoch (other parity) while the first plane reduces this
// one -- the emulated peers running one epoch ahead, which is as far ahead as
// two slots allow. The planes touch disjoint slots and stamps.
//
// The arguments both planes need first come as the kernel's leading scalar
// arguments: gfx950 can preload leading kernel arguments into scalar
// registers when a wave starts (the build asks the compiler for it), so the
// epoch's location and the slot and stamp addresses are known without a
// memory round trip. `shape` packs hidden (bits 0-16), chunks per token (bits
// 17-24), the consumer's slot parity (bit 25) and log2 of the waves per
// workgroup (bits 26-28). The structs carry the rest, read later.
template <int N, int MODE, bool EPI, bool FUSED>
__global__ __launch_bounds__(1024) void reduce_kernel(const uint32_t *ep_base, uint16_t *slots,
                                                      uint32_t *stamps, uint64_t slot_elems,
                                                      uint32_t shape, uint32_t w_max,
                                                      uint32_t ep_off, ReduceArgs ra,
                                                      ProduceArgs pa) {
    const int hidden = static_cast<int>(shape & 0x1FFFFu);
    const int segs = static_cast<int>((shape >> 17) & 0xFFu);
    const int G = 1 << ((shape >> 26) & 7u);
    if (FUSED && blockIdx.z == 1) {
        ProduceArgs pp = pa;
        pp.geo.hidden = hidden;
        pp.geo.segs = segs;
        pp.geo.w_max = static_cast<int32_t>(w_max);
        pp.geo.slot_elems = slot_elems;
        pp.ep.base = ep_base;
        pp.slots = slots;
        pp.stamps = stamps;
        produce_chunk<N>(pp, G);
        return;
    }
    ReduceArgs a = ra;
    a.geo.hidden = hidden;
    a.geo.segs = segs;
    a.geo.w_max = static_cast<int32_t>(w_max);
    a.geo.slot_elems = slot_elems;
    a.ep.base = ep_base;
    a.ep.off = ep_off;
    a.ep.parity = (shape >> 25) & 1u;
    a.slots = slots;
    a.stamps = stamps;
    const int lane = threadIdx.x & (kLanes - 1);
    const int wave = threadIdx.x / kLanes;
    const Geometry &geo = a.geo;
    // The epoch base is read first: its address is at hand, and a uniform
    // load ahead of anything that may write memory stays a scalar load.
    const uint32_t base_v = ep_base[0];
    // grid: x = chunk groups of a token, y = token
    const Chunk k = chunk_at(geo, blockIdx.y, blockIdx.x * G + wave, lane);
    if (!EPI && !k.active) return;  // EPI: idle waves still join the barriers
    const uint32_t p = a.ep.parity;

    V16 rv, wv;
    if (EPI) {
        rv = ld16(a.residual + k.row);
        wv = ld16(a.weight + k.elem);
    }
    V16 v[N];
    uint32_t attempts, first, last, st_first, st_last;
    const uint32_t g =
        gather<N, MODE, true>(a, k, base_v, p, lane, v, attempts, first, last, st_first, st_last);
    const V16 o = sum_round<N>(v);
    if (k.active && lane == 0) {
        write_log(a, k, g, log_word(attempts, first, last));
        a.consumed[static_cast<size_t>(p) * geo.w_max + k.c] = g;
    }
    if (a.stamp_log && k.active && lane < N) write_stamp_log<N>(a, k, g, lane, st_first, st_last);
    if (!EPI) {
        if (k.lane_ok) st16_stream(a.out + k.row, o);
        return;
    }
    residual_rmsnorm(a, k, g, o, rv, wv, a.y, lane, wave, G, blockIdx.x);
}

// The persistent step's epilogue in two halves, so that the wait for the
// token's other groups overlaps the next epoch's reduction instead of
// stalling every chunk of the token once per epoch. Only the residual carries
// from one epoch to the next, and it is this chunk's own; the token-wide sum of
// squares is needed for y alone. epi_stage runs right after epoch g's sum: it
// updates the residual, reduces this group's sum of squares and publishes it
// in exchange plane g mod kExchPlanes. epi_finish runs one epoch later, or
// after the step's last epoch: it waits for the token's Q words of epoch g,
// adds them in group order and writes y. The arithmetic and its order are
// residual_rmsnorm's. Four planes suffice: a group can publish epoch g + 4
// only after finishing epoch g + 2, which needs every group's word of g + 2,
// and a group publishes that only after it finished epoch g.
struct EpiPending {
    float x[kVec];  // res' of this lane's 8 elements, widened to fp32
    float grp;      // this workgroup's sum of squares
    uint32_t g;     // the epoch
};

__device__ __forceinline__ void epi_stage(const ReduceArgs &a, const Chunk &k, uint32_t g,
                                          const V16 &o, const V16 &rv, int lane, int wave, int G,
                                          int q, bool xlocal, EpiPending &pd) {
    V16 nr;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float a0 = lo_f32(o.w[i]), a1 = hi_f32(o.w[i]);
        nr.w[i] = pack_bf16(a0 + lo_f32(rv.w[i]), a1 + hi_f32(rv.w[i]));
        pd.x[2 * i] = lo_f32(nr.w[i]);
        pd.x[2 * i + 1] = hi_f32(nr.w[i]);
    }
    if (k.lane_ok) st16(a.residual + k.row, nr);

    float ss = 0.f;
    if (k.lane_ok) {
#pragma unroll
        for (int i = 0; i < kVec; ++i) ss = __builtin_fmaf(pd.x[i], pd.x[i], ss);
    }
#pragma unroll
    for (int off = kLanes / 2; off >= 1; off >>= 1) ss = ss + __shfl_xor(ss, off);

    __shared__ float part[kMaxWavesPerGroup];
    if (lane == 0) part[wave] = ss;
    __syncthreads();
    float grp = 0.f;
    for (int w = 0; w < G; ++w) grp = grp + part[w];
    pd.grp = grp;
    pd.g = g;

    const int Q = a.groups_per_token;
    if (Q > 1 && wave == 0 && lane == 0) {
        uint64_t *ex = a.exch + static_cast<size_t>(g % kExchPlanes) * a.exch_parity_stride +
                       static_cast<size_t>(k.t) * Q;
        const uint64_t word = (static_cast<uint64_t>(g) << 32) | __float_as_uint(grp);
        // all groups of the token on this XCD: the word meets them in its L2
        if (xlocal)
            __hip_atomic_store(ex + q, word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        else
            __hip_atomic_store(ex + q, word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// `y` is the ring entry of epoch pd.g. (`pd` by value: with a reference the
// compiler kept the pending state in scratch memory.) True in wave 0 when the
// exchange wait failed: it ran out of polls (latched here), or found an error
// latched elsewhere.
__device__ __forceinline__ bool epi_finish(const ReduceArgs &a, const Chunk &k,
                                           const EpiPending pd, const V16 &wv, uint16_t *y,
                                           int lane, int wave) {
    const int Q = a.groups_per_token;
    float tot = pd.grp;
    bool failed = false;
    if (Q > 1) {
        __shared__ float total;
        if (wave == 0) {
            const uint64_t *ex = a.exch +
                                 static_cast<size_t>(pd.g % kExchPlanes) * a.exch_parity_stride +
                                 static_cast<size_t>(k.t) * Q;
            uint64_t mine = 0;
            uint32_t spins = 0;
            bool ready;
            do {
                if (lane < Q)
                    mine = __hip_atomic_load(ex + lane, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                ready = __ballot(lane < Q && static_cast<uint32_t>(mine >> 32) != pd.g) == 0;
                if (!ready && spins >= kErrPollAfter && ld_relaxed(a.err) != 0) break;
            } while (!ready && ++spins < a.spin_limit);
            failed = !ready;
            if (!ready && lane == 0) latch(a.err, kErrExchange, pd.g, k.c, spins);
            const float pv = __uint_as_float(static_cast<uint32_t>(mine));
            float sum = 0.f;
            for (int j = 0; j < Q; ++j) sum = sum + __shfl(pv, j);
            if (lane == 0) total = sum;
        }
        __syncthreads();
        tot = total;
    }
    const float inv = 1.0f / __builtin_sqrtf(tot / static_cast<float>(a.geo.hidden) + a.eps);
    V16 yo;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float w0 = lo_f32(wv.w[i]), w1 = hi_f32(wv.w[i]);
        yo.w[i] = pack_bf16((pd.x[2 * i] * inv) * w0, (pd.x[2 * i + 1] * inv) * w1);
    }
    if (k.lane_ok) st16(y + k.row, yo);
    return failed;
}

// ---------------------------------------------------------------------------
// Persistent decode step: one launch runs all L all-reduces. All waves are
// co-resident (the host checks), and every wait is bounded.
//
// Per chunk and epoch g of parity p:
//   producer  wait until consumed[p] == produced[p] (the reduction that read
//             this slot two epochs back has finished: dual buffering), copy
//             the N partials, publish them (publish_slot: a release fence
//             only when the consumer is on another XCD), store the on-time
//             stamps and produced[p] = g; injected late ranks' stamps follow
//             after `late_delay` sleeps.
//   consumer  poll the stamps (relaxed agent-scope loads, back to back) until
//             all are fresh, then load the payload (after an acquire fence
//             when the producer is on another XCD); sum; store; consumed[p] =
//             g once every payload load has completed.
// Every wait is bounded, and joins the error word to its polls only once it
// has lasted kErrPollAfter polls.
// Validation comes before the payload loads here (ORDERED). Speculative
// payload loads issued alongside the stamp loads were measured to return a
// rank's previous epoch while its stamp already read as fresh when producer
// and consumer sat on different XCDs: the monotonicity the paper assumes
// (Sec. 8.1) does not hold for a live producer on MI355X. (The per-epoch
// launches keep SPEC: there every epoch was written by an earlier launch.)
// The producer can run one epoch ahead of the consumer, no further.
// Producer wave of chunk (t, s), one epoch after the other: wait until the
// slot of this parity is free (with a single buffer: until the previous
// epoch's reduction is done -- the bottom barrier), store the sources already
// in registers, publish, stamps. Loading the next epoch's sources while the
// slot stores travel shortened the llama8b decode step by ~5 % on MI355X once
// the consumer issued its polls ahead of its stores; before that the consumer
// bounded the step and the prefetch made no difference.
template <int N, bool PREFETCH>
__device__ __forceinline__ void chain_producer(const ChainArgs &A, uint32_t base, int lane,
                                               int bx, int by) {
    const ProduceArgs &a = A.p;
    const Geometry &geo = a.geo;
    const Chunk k = chunk_at(geo, by, bx, lane);
    publish_place(A.place + geo.w_max + k.c, base, lane);
    const bool local = partner_is_local(A.place + k.c, base, lane);
    // One epoch: wait until the slot is free, store `cur` (the epoch's
    // sources, already in registers), load the next epoch's sources into
    // `nxt` while the slot stores travel (harmless in-bounds reads after the
    // last epoch), publish, stamp. False when the slot wait failed.
    auto epoch = [&](int i, const V16(&cur)[N], V16(&nxt)[N]) -> bool {
        const uint32_t g = base + static_cast<uint32_t>(i) + 1u;
        const uint32_t p = static_cast<uint32_t>(i + 1) & A.parity_mask;
        const size_t pc = static_cast<size_t>(p) * geo.w_max + k.c;
        uint32_t spins = 0;
        bool free = false;
        // one round trip per poll: both words together, and the error word
        // after kErrPollAfter polls; a short sleep between polls (without it
        // the kernel takes 109 VGPRs instead of 76 and the step ran ~0.6 %
        // slower)
        while (true) {
            const uint32_t done = ld_relaxed(a.consumed + pc);
            const uint32_t prev = ld_relaxed(a.produced + pc);
            const uint32_t e = spins >= kErrPollAfter ? ld_relaxed(a.err) : 0u;
            free = done == prev;
            if (free || ++spins >= A.r.spin_limit || e != 0) break;
            __builtin_amdgcn_s_sleep(1);
        }
        if (!free) {
            if (lane == 0) latch(a.err, kErrWaw, g, k.c, spins);
            return false;
        }
        const uint32_t inj = inject_word(a.inject, a.inject_div, g);
        const uint32_t held = held_back(inj);
        if (!PREFETCH) {
            copy_chunk<N>(a, k, g, p);
            publish_slot(local);
        } else if (local) {
            store_slots_at<N>(a, k, p, cur);
            // the loads stay after the stores (the wait below counts on it)
            __atomic_signal_fence(__ATOMIC_SEQ_CST);
            load_sources<N>(a, k, g + 1u, nxt);
            // Loads and stores complete in issue order on gfx9-family GPUs:
            // with at most N operations outstanding the slot stores have
            // reached the L2 and only the N source loads are still in flight.
            __builtin_amdgcn_s_waitcnt(kWaitVm | N);
            __atomic_signal_fence(__ATOMIC_SEQ_CST);
        } else {
            store_slots_at<N>(a, k, p, cur);
            load_sources<N>(a, k, g + 1u, nxt);
            publish_slot(false);
        }
        uint32_t *stamp = a.stamps + pc * N;
        if (lane < N && !((held >> lane) & 1u)) st_flag(stamp + lane, g, local);
        if (lane == 0) st_flag(a.produced + pc, g, local);
        if (held) {
            for (uint32_t d = 0; d < A.late_delay; ++d) __builtin_amdgcn_s_sleep(8);
            if (lane < N && ((inj >> lane) & 1u) && !((inj >> (8 + lane)) & 1u))
                st_flag(stamp + lane, g, local);
        }
        return true;
    };
    // Two register sets taking turns: a load never overwrites the data of a
    // store still in flight, so nothing waits for the store acknowledgements
    // before the next sources are requested. (Without PREFETCH every epoch
    // loads and stores in one go: 2N fewer registers, for steps whose waves
    // fit on the GPU only at the higher occupancy.)
    V16 va[N], vb[N];
    if (PREFETCH) load_sources<N>(a, k, base + 1u, va);
    for (int i = 0; i < A.reduces; i += 2) {
        if (!epoch(i, va, vb)) return;
        if (i + 1 < A.reduces && !epoch(i + 1, vb, va)) return;
    }
}

// Grouped producer of epilogue steps (G waves per workgroup, one chunk per
// wave): the waves
// copy their chunks, wait until their stores have reached L2, meet at a
// workgroup barrier, and wave 0 publishes for all of them (one agent-scope
// release fence, needed only when a consumer of the group is on another XCD)
// and stores every chunk's stamps (lane = chunk wave * N + rank). Such fences
// write back the XCD's L2 and serialise per XCD, so sharing one among G chunks
// shortens the epoch once several producer waves share each XCD. Every wave
// reaches the barrier in every epoch; a failed slot wait ends the whole
// workgroup at the same barrier.
template <int N>
__device__ __forceinline__ void chain_producer_grouped(const ChainArgs &A, uint32_t base,
                                                       int lane, int wave, int G, int bx, int by) {
    const ProduceArgs &a = A.p;
    const Geometry &geo = a.geo;
    const Chunk k = chunk_at(geo, by, bx * G + wave, lane);
    const int sw = lane / N, sr = lane - sw * N;
    const Chunk ks = chunk_at(geo, by, bx * G + (sw < G ? sw : 0), 0);
    const bool stamper = wave == 0 && sw < G && ks.active;
    if (k.active) publish_place(A.place + geo.w_max + k.c, base, lane);
    const bool mine = !k.active || partner_is_local(A.place + k.c, base, lane);
    const bool local = __syncthreads_and(mine ? 1 : 0) != 0;
    for (int i = 0; i < A.reduces; ++i) {
        const uint32_t g = base + static_cast<uint32_t>(i) + 1u;
        const uint32_t p = static_cast<uint32_t>(i + 1) & A.parity_mask;
        bool free = true;
        if (k.active) {
            const size_t pc = static_cast<size_t>(p) * geo.w_max + k.c;
            uint32_t spins = 0;
            while (true) {  // one round trip per poll, as in chain_producer
                const uint32_t done = ld_relaxed(a.consumed + pc);
                const uint32_t prev = ld_relaxed(a.produced + pc);
                const uint32_t e = spins >= kErrPollAfter ? ld_relaxed(a.err) : 0u;
                free = done == prev;
                if (free || ++spins >= A.r.spin_limit || e != 0) break;
                __builtin_amdgcn_s_sleep(1);
            }
            if (!free && lane == 0) latch(a.err, kErrWaw, g, k.c, spins);
            if (free) {
                copy_chunk<N>(a, k, g, p);
                // only this wave reads its chunk's produced word: recording it
                // here, not after wave 0's fence, keeps the next epoch's slot
                // check from seeing the previous value (with one buffer that
                // would let the slot be rewritten before it is consumed)
                if (lane == 0) st_flag(a.produced + pc, g, true);
            }
        }
        __builtin_amdgcn_s_waitcnt(0);  // this wave's slot stores have reached L2
        if (__syncthreads_or(!free)) return;
        if (wave == 0) {
            const uint32_t inj = inject_word(a.inject, a.inject_div, g);
            const uint32_t held = held_back(inj);
            publish_slot(local);  // with `local` the wait above already did it
            const size_t ps = static_cast<size_t>(p) * geo.w_max + ks.c;
            uint32_t *stamp = a.stamps + ps * N;
            if (stamper && !((held >> sr) & 1u)) st_flag(stamp + sr, g, local);
            if (held) {
                for (uint32_t d = 0; d < A.late_delay; ++d) __builtin_amdgcn_s_sleep(8);
                if (stamper && ((inj >> sr) & 1u) && !((inj >> (8 + sr)) & 1u))
                    st_flag(stamp + sr, g, local);
            }
        }
    }
}

// Consumer wave of chunk (t, x * G + wave). With G > 1 and the epilogue the
// group's waves share the RMSNorm barriers, so they also leave together.
template <int N, int MODE, bool EPI, bool GROUPED>
__device__ __forceinline__ void chain_consumer(const ChainArgs &A, uint32_t base, int lane,
                                               int wave, int G, int bx, int by) {
    const ReduceArgs &a = A.r;
    const Geometry &geo = a.geo;
    const Chunk k = chunk_at(geo, by, bx * G + wave, lane);
    if (k.active) publish_place(A.place + k.c, base, lane);
    const bool local = k.active && partner_is_local(A.place + geo.w_max + k.c, base, lane);
    // the epilogue's exchange partners: wave 0 of each group of this token
    bool xlocal = false;
    if (EPI && wave == 0) {
        const int Q = a.groups_per_token;
        const bool mine = lane >= Q ||
                          tag_is_local(A.place + static_cast<size_t>(k.t) * geo.segs + lane * G, base);
        xlocal = __ballot(!mine) == 0;
    }
    V16 wv;
    if (EPI) wv = ld16(a.weight + k.elem);
    EpiPending pending;   // the epilogue of the previous epoch, finished one epoch late
    bool have_pending = false;
    // Every lane polls a stamp of this chunk (lanes >= N repeat rank N - 1's,
    // which the ballot ignores), so no branch surrounds the poll.
    const uint32_t *stamps = a.stamps + static_cast<size_t>(k.c) * N + (lane < N ? lane : N - 1);
    const size_t parity_stride = static_cast<size_t>(geo.w_max) * N;
    // The first poll of an epoch -- its stamps -- is issued before the
    // previous epoch's stores. On gfx9-family GPUs one counter
    // (vmcnt) tracks loads and stores in issue order, so a poll issued after
    // the stores could only be waited for together with their write
    // acknowledgements. The stores below are therefore branch-free too, so the
    // compiler can count them and wait for the poll alone. An early poll that
    // reads stale is repeated; the payload is still loaded only after fresh
    // stamps were seen.
    uint32_t st_next = ld_relaxed(stamps + (1u & A.parity_mask) * parity_stride);
    // stale ranks of the first poll, evaluated where the wait for it is exact
    uint32_t m_next = static_cast<uint32_t>(__ballot(lane < N && st_next != base + 1u));
    for (int i = 0; i < A.reduces; ++i) {
        const uint32_t g = base + static_cast<uint32_t>(i) + 1u;
        const uint32_t p = static_cast<uint32_t>(i + 1) & A.parity_mask;
        V16 rv;
        if (EPI) rv = ld16(a.residual + k.row);  // this wave's own previous store
        V16 v[N];
        uint32_t attempts, first, last;
        const uint32_t st_first = st_next;
        uint32_t st_last = st_next;
        bool stop =
            gather_chain<N, !EPI>(a, k, g, p, lane, m_next, st_last, v, attempts, first, last, local);
        uint32_t *consumed = a.consumed + static_cast<size_t>(p) * geo.w_max + k.c;
        // Once the payload has arrived: issue the next epoch's first poll (a
        // harmless in-bounds read after the last epoch), then release the slot
        // (every lane stores the same word).
        auto poll_next_and_release = [&]() {
            const uint32_t pn = static_cast<uint32_t>(i + 2) & A.parity_mask;
            st_next = ld_relaxed(stamps + pn * parity_stride);
            __atomic_signal_fence(__ATOMIC_SEQ_CST);  // keep the poll ahead of the stores
            st_flag(consumed, g, local);
        };
        if (!EPI) {
            // release the slot as soon as every payload load has returned (the
            // sum works on registers); measured faster for the plain chain,
            // slower with the epilogue
#pragma unroll
            for (int r = 0; r < N; ++r) complete(v[r]);
            poll_next_and_release();
        }
        const V16 o = sum_round<N>(v);
        if (EPI) {
            complete(o);  // every payload load has returned before the slot is released
            poll_next_and_release();
        }
        write_log(a, k, g, log_word(attempts, first, last));  // wave-uniform word
        // lanes >= N store rank N - 1's stamps again: the same words to the same place
        write_stamp_log<N>(a, k, g, lane < N ? lane : N - 1, st_first, st_last);
        const uint64_t ring = static_cast<uint64_t>(i) * A.ring_stride;
        if (!EPI) {
            // Lanes past the end of the row loaded the row's last 8 elements
            // (clamped) with the same instruction as the lane that owns them,
            // so they store the same bytes to the same place: no branch.
            st16_stream(a.out + ring + k.row, o);
        } else {
            EpiPending cur;
            epi_stage(a, k, g, o, rv, lane, wave, G, bx, xlocal, cur);
            if (have_pending &&
                epi_finish(a, k, pending, wv, a.y + ring - A.ring_stride, lane, wave))
                stop = true;
            pending = cur;
            have_pending = true;
        }
        // The next epoch's first poll, after this epoch's stores: the
        // compiler waits for the poll alone and leaves the stores in flight.
        m_next = static_cast<uint32_t>(__ballot(lane < N && st_next != g + 1u));
        // a bounded wait of this wave failed: stop (a pending epilogue stays
        // unwritten: the step has failed). Every wait is bounded and reads the
        // error word once it has lasted kErrPollAfter polls, so a failure
        // anywhere ends the other waves' waits too.
        if (GROUPED && EPI) {
            if (__syncthreads_or(stop)) return;
        } else if (stop) {
            return;
        }
    }
    if (EPI && have_pending)
        epi_finish(a, k, pending, wv, a.y + static_cast<uint64_t>(A.reduces - 1) * A.ring_stride,
                   lane, wave);
}

// Grid (segs, tokens, 2) of one-wave workgroups, or with the epilogue
// (8 * ceil(tokens / 8) * Q, 1, 2) of G-wave workgroups (G = 1, or
// kChainGroupWaves when GROUPED; Q = segs / G, layout below): plane 0 reduces
// chunk (t, x * G + wave) for epochs base+1 .. base+L in order, plane 1
// produces it. The last wave to arrive on the counter advances the epoch base
// for the next step: every wave read the base before it arrived, so no wave
// can see the advanced value.
template <int N, int MODE, bool EPI, bool GROUPED, bool PREFETCH>
__global__ __launch_bounds__(GROUPED ? kChainGroupWaves * kLanes : kLanes,
                             1) void chain_kernel(ChainArgs A) {
    const int lane = threadIdx.x & (kLanes - 1);
    const int wave = GROUPED ? static_cast<int>(threadIdx.x) / kLanes : 0;
    const int G = GROUPED ? static_cast<int>(blockDim.x) / kLanes : 1;
    const uint32_t base = A.r.ep.base[0];
    // Logical (group, token). With the epilogue, workgroup b of a plane serves
    // token (b mod 8) + 8 * (b / 8 / Q), group (b / 8) mod Q: every group of a
    // token -- consumers and producers, since each plane holds a multiple of 8
    // workgroups -- is dealt to the same XCD, so the per-epoch exchange of the
    // token's sum of squares stays in one L2. Workgroups past the last token
    // only arrive on the counter.
    int bx = blockIdx.x, by = blockIdx.y;
    if (EPI) {
        const int Q = A.r.groups_per_token;
        const int j = static_cast<int>(blockIdx.x) >> 3;
        bx = j % Q;
        by = (static_cast<int>(blockIdx.x) & 7) + 8 * (j / Q);
    }
    if (by < A.r.geo.tokens) {
        if (blockIdx.z == 1) {
            if (GROUPED)
                chain_producer_grouped<N>(A, base, lane, wave, G, bx, by);
            else
                chain_producer<N, PREFETCH>(A, base, lane, bx, by);
        } else {
            chain_consumer<N, MODE, EPI, GROUPED>(A, base, lane, wave, G, bx, by);
        }
    }
    if (lane == 0) {
        const uint32_t waves = 2u * gridDim.x * gridDim.y * static_cast<uint32_t>(G);
        const uint32_t before =
            __hip_atomic_fetch_add(A.done, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (before == waves - 1u) {
            st_relaxed(A.done, 0u);
            st_relaxed(A.epoch_base, base + A.advance);
        }
    }
}

__global__ void advance_kernel(uint32_t *base, uint32_t step) {
    if (threadIdx.x == 0) base[0] += step;
}

__global__ void set_base_kernel(uint32_t *base, uint32_t value) {
    if (threadIdx.x == 0) base[0] = value;
}

__global__ void fill_u32_kernel(uint32_t *p, uint32_t value, uint64_t count) {
    for (uint64_t i = blockIdx.x * static_cast<uint64_t>(blockDim.x) + threadIdx.x; i < count;
         i += static_cast<uint64_t>(gridDim.x) * blockDim.x)
        p[i] = value;
}

template <int N, int MODE>
hipError_t launch_reduce_nm(const ReduceArgs &a, const ProduceArgs *pa, bool epi, dim3 grid,
                            dim3 block, hipStream_t s) {
    const ProduceArgs none{};
    int lg = 0;
    while ((kLanes << lg) < static_cast<int>(block.x)) ++lg;
    if ((kLanes << lg) != static_cast<int>(block.x) || lg > 4) return hipErrorInvalidValue;
    if (a.geo.hidden < 1 || a.geo.hidden > 0x10000 || a.geo.segs < 1 || a.geo.segs > 0xFF ||
        a.ep.parity > 1)
        return hipErrorInvalidValue;
    // the producer plane shares the leading arguments (one handle's slots,
    // stamps, epoch and geometry)
    if (pa && (pa->ep.base != a.ep.base || pa->slots != a.slots || pa->stamps != a.stamps ||
               pa->geo.hidden != a.geo.hidden || pa->geo.w_max != a.geo.w_max ||
               pa->geo.slot_elems != a.geo.slot_elems))
        return hipErrorInvalidValue;
    const uint32_t shape = static_cast<uint32_t>(a.geo.hidden) |
                           (static_cast<uint32_t>(a.geo.segs) << 17) | (a.ep.parity << 25) |
                           (static_cast<uint32_t>(lg) << 26);
    const uint32_t w_max = static_cast<uint32_t>(a.geo.w_max);
#define SIFAR_REDUCE_LAUNCH(EPI_, FUSED_, PA_)                                                   \
    hipLaunchKernelGGL((reduce_kernel<N, MODE, EPI_, FUSED_>), grid, block, 0, s, a.ep.base,   \
                       a.slots, a.stamps, a.geo.slot_elems, shape, w_max, a.ep.off, a, PA_)
    if (pa) {
        grid.z = 2;
        if (epi)
            SIFAR_REDUCE_LAUNCH(true, true, *pa);
        else
            SIFAR_REDUCE_LAUNCH(false, true, *pa);
    } else {
        if (epi)
            SIFAR_REDUCE_LAUNCH(true, false, none);
        else
            SIFAR_REDUCE_LAUNCH(false, false, none);
    }
#undef SIFAR_REDUCE_LAUNCH
    return hipGetLastError();
}

template <int N>
hipError_t launch_reduce_n(const ReduceArgs &a, const ProduceArgs *pa, int mode, bool epi,
                           dim3 grid, dim3 block, hipStream_t s) {
    switch (mode) {
        case kSpec: return launch_reduce_nm<N, kSpec>(a, pa, epi, grid, block, s);
        case kOrdered: return launch_reduce_nm<N, kOrdered>(a, pa, epi, grid, block, s);
        case kNone: return launch_reduce_nm<N, kNone>(a, pa, epi, grid, block, s);
    }
    return hipErrorInvalidValue;
}

// Grouped workgroups serve epilogue steps only (plain steps measured faster
// or level with one wave per workgroup); the grouped producer loads and
// stores in one go. With the epilogue the consumer sets the register count,
// so only the plain one-wave-per-chunk kernel comes in both producer forms.
template <int N, int MODE>
const void *chain_fn(bool epi, bool grouped, bool prefetch) {
    if (grouped)
        return epi ? reinterpret_cast<const void *>(chain_kernel<N, MODE, true, true, false>)
                   : nullptr;
    if (epi) return reinterpret_cast<const void *>(chain_kernel<N, MODE, true, false, true>);
    return prefetch ? reinterpret_cast<const void *>(chain_kernel<N, MODE, false, false, true>)
                    : reinterpret_cast<const void *>(chain_kernel<N, MODE, false, false, false>);
}

// Persistent steps validate before they load: ORDERED only.
template <int N>
const void *chain_fn_n(int mode, bool epi, bool grouped, bool prefetch) {
    return mode == kOrdered ? chain_fn<N, kOrdered>(epi, grouped, prefetch) : nullptr;
}

const void *chain_fn_any(int nranks, int mode, bool epi, bool grouped, bool prefetch) {
    switch (nranks) {
        case 1: return chain_fn_n<1>(mode, epi, grouped, prefetch);
        case 2: return chain_fn_n<2>(mode, epi, grouped, prefetch);
        case 3: return chain_fn_n<3>(mode, epi, grouped, prefetch);
        case 4: return chain_fn_n<4>(mode, epi, grouped, prefetch);
        case 5: return chain_fn_n<5>(mode, epi, grouped, prefetch);
        case 6: return chain_fn_n<6>(mode, epi, grouped, prefetch);
        case 7: return chain_fn_n<7>(mode, epi, grouped, prefetch);
        case 8: return chain_fn_n<8>(mode, epi, grouped, prefetch);
    }
    return nullptr;
}

template <int N, int MODE>
const void *reduce_fn(bool epi) {
    // the fused variant is the larger of the two: use it for occupancy
    return epi ? reinterpret_cast<const void *>(reduce_kernel<N, MODE, true, true>)
               : reinterpret_cast<const void *>(reduce_kernel<N, MODE, false, true>);
}

template <int N>
const void *reduce_fn_n(int mode, bool epi) {
    switch (mode) {
        case kSpec: return reduce_fn<N, kSpec>(epi);
        case kOrdered: return reduce_fn<N, kOrdered>(epi);
        case kNone: return reduce_fn<N, kNone>(epi);
    }
    return nullptr;
}

const void *reduce_fn_any(int nranks, int mode, bool epi) {
    switch (nranks) {
        case 1: return reduce_fn_n<1>(mode, epi);
        case 2: return reduce_fn_n<2>(mode, epi);
        case 3: return reduce_fn_n<3>(mode, epi);
        case 4: return reduce_fn_n<4>(mode, epi);
        case 5: return reduce_fn_n<5>(mode, epi);
        case 6: return reduce_fn_n<6>(mode, epi);
        case 7: return reduce_fn_n<7>(mode, epi);
        case 8: return reduce_fn_n<8>(mode, epi);
    }
    return nullptr;
}

int resident_groups(const void *fn, int threads) {
    if (!fn) return 0;
    int per_cu = 0, dev = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, threads, 0) != hipSuccess)
        return 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return 0;
    return per_cu * cus;
}

}  // namespace

hipError_t launch_produce(const ProduceArgs &a, int waves_per_group, hipStream_t s) {
    const dim3 grid(static_cast<uint32_t>((a.geo.segs + waves_per_group - 1) / waves_per_group),
                    static_cast<uint32_t>(a.geo.tokens));
    const dim3 block(waves_per_group * kLanes);
    switch (a.geo.nranks) {
        case 1: hipLaunchKernelGGL(produce_kernel<1>, grid, block, 0, s, a); break;
        case 2: hipLaunchKernelGGL(produce_kernel<2>, grid, block, 0, s, a); break;
        case 3: hipLaunchKernelGGL(produce_kernel<3>, grid, block, 0, s, a); break;
        case 4: hipLaunchKernelGGL(produce_kernel<4>, grid, block, 0, s, a); break;
        case 5: hipLaunchKernelGGL(produce_kernel<5>, grid, block, 0, s, a); break;
        case 6: hipLaunchKernelGGL(produce_kernel<6>, grid, block, 0, s, a); break;
        case 7: hipLaunchKernelGGL(produce_kernel<7>, grid, block, 0, s, a); break;
        case 8: hipLaunchKernelGGL(produce_kernel<8>, grid, block, 0, s, a); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_reduce(const ReduceArgs &a, const ProduceArgs *next, int mode, bool epilogue,
                         int waves_per_group, hipStream_t s) {
    const dim3 block(waves_per_group * kLanes);
    const dim3 grid(static_cast<uint32_t>((a.geo.segs + waves_per_group - 1) / waves_per_group),
                    static_cast<uint32_t>(a.geo.tokens));
    if (next && (next->geo.segs != a.geo.segs || next->geo.tokens != a.geo.tokens))
        return hipErrorInvalidValue;
    switch (a.geo.nranks) {
        case 1: return launch_reduce_n<1>(a, next, mode, epilogue, grid, block, s);
        case 2: return launch_reduce_n<2>(a, next, mode, epilogue, grid, block, s);
        case 3: return launch_reduce_n<3>(a, next, mode, epilogue, grid, block, s);
        case 4: return launch_reduce_n<4>(a, next, mode, epilogue, grid, block, s);
        case 5: return launch_reduce_n<5>(a, next, mode, epilogue, grid, block, s);
        case 6: return launch_reduce_n<6>(a, next, mode, epilogue, grid, block, s);
        case 7: return launch_reduce_n<7>(a, next, mode, epilogue, grid, block, s);
        case 8: return launch_reduce_n<8>(a, next, mode, epilogue, grid, block, s);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_chain(const ChainArgs &a, int mode, bool epilogue, int waves, bool prefetch,
                        hipStream_t s) {
    if (waves != 1 && waves != kChainGroupWaves) return hipErrorInvalidValue;
    const void *fn = chain_fn_any(a.r.geo.nranks, mode, epilogue, waves > 1, prefetch);
    if (!fn) return hipErrorInvalidValue;
    if (a.r.geo.segs != a.p.geo.segs || a.r.geo.tokens != a.p.geo.tokens ||
        a.r.geo.segs % waves != 0 || (waves > 1 && waves * a.r.geo.nranks > kLanes))
        return hipErrorInvalidValue;
    const uint32_t q = static_cast<uint32_t>(a.r.geo.segs / waves);
    const uint32_t t8 = (static_cast<uint32_t>(a.r.geo.tokens) + 7u) / 8u;
    if (epilogue && a.r.groups_per_token != static_cast<int32_t>(q)) return hipErrorInvalidValue;
    // the slots are addressed at 32-bit offsets from rank 0's (payload loads,
    // slot stores); co-residency keeps a step far below that (at most 4096
    // chunks: under 64 MiB of slots)
    if (static_cast<uint64_t>(a.r.geo.nranks) * 4u * a.r.geo.slot_elems > 0x7fffffffull)
        return hipErrorInvalidValue;
    const dim3 grid = epilogue ? dim3(8u * t8 * q, 1, 2)
                               : dim3(q, static_cast<uint32_t>(a.r.geo.tokens), 2);
    void *args[] = {const_cast<ChainArgs *>(&a)};
    return hipLaunchKernel(fn, grid, dim3(kLanes * waves), args, 0, s);
}

int max_active_groups(int nranks, int mode, bool epilogue, int waves_per_group) {
    return resident_groups(reduce_fn_any(nranks, mode, epilogue), waves_per_group * kLanes);
}

int max_active_chain_groups(int nranks, int mode, bool epilogue, int waves, bool prefetch) {
    if (waves != 1 && waves != kChainGroupWaves) return 0;
    return resident_groups(chain_fn_any(nranks, mode, epilogue, waves > 1, prefetch),
                           waves * kLanes);
}

hipError_t launch_advance(uint32_t *epoch_base, uint32_t step, hipStream_t s) {
    hipLaunchKernelGGL(advance_kernel, dim3(1), dim3(kLanes), 0, s, epoch_base, step);
    return hipGetLastError();
}

hipError_t launch_set_base(uint32_t *epoch_base, uint32_t value, hipStream_t s) {
    hipLaunchKernelGGL(set_base_kernel, dim3(1), dim3(kLanes), 0, s, epoch_base, value);
    return hipGetLastError();
}

hipError_t launch_fill_u32(uint32_t *p, uint32_t value, uint64_t count, hipStream_t s) {
    if (count == 0) return hipSuccess;
    const uint64_t blocks64 = (count + 255) / 256;
    const dim3 grid(static_cast<uint32_t>(blocks64 < 4096 ? blocks64 : 4096));
    hipLaunchKernelGGL(fill_u32_kernel, grid, dim3(256), 0, s, p, value, count);
    return hipGetLastError();
}

}  // namespace sifar
