// Message-passing litmus of the handoff a persistent decode step runs between
// the emulated peers and the reduction: one producer wave and one consumer
// wave pass a dual-buffered slot (8 ranks x 64 lanes x 16 bytes, the size of
// one chunk) back and forth for many epochs, with the same primitives and the
// same slot discipline as the all-reduce (a slot of parity g & 1 is rewritten
// only after its previous epoch was consumed, Sec. 3.3 and 4.1), and the
// consumer checks every word it accepted against the epoch it validated.
//
// Two reader orders:
//  - ORDERED, the persistent step's: poll the stamps until all are fresh, then
//    acquire (only from another XCD), then load the payload;
//  - READ_FIRST, the paper's speculative order (Sec. 4.2): load payload and
//    stamps together, accept when every stamp is fresh, else acquire and
//    reload both.
// Two producer forms: the plain one stores the slot and waits for every
// outstanding operation (publish_slot); the prefetching one publishes as the
// persistent step's prefetching producer does -- buffer stores of the slot,
// then buffer loads of the next epoch's sources, then a wait until at most
// those loads are outstanding (vmcnt(8)), then the flags -- so the ordering
// that wait relies on (one wave's vector memory operations leave the counter
// in issue order) is checked on the sequence the benchmark's kernel runs.
// Pairs are laid out so that, with workgroups dealt to the XCDs round robin,
// producer and consumer sit on different XCDs (or on the same one); each wave
// reads its XCC_ID and the pair reports whether it landed as intended, and the
// handoff itself takes the partner's real placement into account. Every wait
// is bounded: a wave that gives up records a timeout and leaves, and its
// partner's next wait then runs out too.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "coherence.h"
#include "sifar.h"

namespace sifar {
namespace {

constexpr int kLitmusRanks = 8;
constexpr int kWaveLanes = 64;
constexpr int kSlotWords = kLitmusRanks * kWaveLanes * 4;  // u32 words per slot
constexpr int kMaxPairs = 512;
constexpr int kMaxTrials = 1 << 20;
constexpr uint32_t kSpins = 1u << 20;  // polls per wait before giving up
constexpr uint32_t kValueStep = 0x9E3779B1u;  // odd: epochs g and g - 2 never share a word value

// per-pair result words
enum {
    O_TRIALS, O_BAD, O_BAD_EARLY, O_TIMEOUT, O_PRODUCER_TIMEOUT, O_PLACED, O_BAD_G, O_BAD_FOUND,
    O_BAD_WANT, O_XCC, O_WORDS
};

struct LitmusArgs {
    uint32_t *slots;     // [pair][parity][rank][lane][4]
    uint32_t *stamps;    // [parity][pair][rank]
    uint32_t *consumed;  // [parity][pair]
    uint32_t *produced;  // [parity][pair]
    uint64_t *place;     // [producer, consumer][pair]
    uint32_t *out;       // [pair][O_WORDS]
    uint64_t *ticks;     // [pair][2]: consumer's start and end
    const uint32_t *src; // [pair][rank][lane][4], all zero: the prefetching producer's sources
    int pairs, trials, read_first, cross, prefetch;
};

// Word w of rank r and lane l in epoch g.
__device__ __forceinline__ uint32_t value_of(uint32_t g, int r, int lane, int w) {
    return g * kValueStep + static_cast<uint32_t>((r * kWaveLanes + lane) * 4 + w);
}

__device__ __forceinline__ uint32_t *slot_of(const LitmusArgs &a, int pair, uint32_t p, int r,
                                             int lane) {
    return a.slots + ((static_cast<size_t>(pair) * 2 + p) * kLitmusRanks + r) * kWaveLanes * 4 +
           lane * 4;
}

// Slot word offset of rank r's 16 bytes for `lane`, from the pair's parity-p
// slot start (the buffer form's per-lane byte offset).
__device__ __forceinline__ uint32_t lane_bytes(int lane) { return static_cast<uint32_t>(lane) * 16u; }

// The prefetching producer: epoch g's slot is stored from values derived from
// sources loaded one epoch earlier (zeros, unknown to the compiler), and the
// next epoch's sources are loaded while the slot stores travel.
__device__ void producer_prefetch(const LitmusArgs &a, int pair, int lane, bool local) {
    const uint32_t *src = a.src + static_cast<size_t>(pair) * kLitmusRanks * kWaveLanes * 4;
    V16 raw[kLitmusRanks];
#pragma unroll
    for (int r = 0; r < kLitmusRanks; ++r)
        raw[r] = ld16_buffer<0>(src + r * kWaveLanes * 4, lane_bytes(lane));
    for (int i = 1; i <= a.trials; ++i) {
        const uint32_t g = static_cast<uint32_t>(i), p = g & 1u;
        const size_t pc = static_cast<size_t>(p) * a.pairs + pair;
        bool free = false;
        for (uint32_t spins = 0; spins < kSpins; ++spins) {
            free = ld_relaxed(a.consumed + pc) == ld_relaxed(a.produced + pc);
            if (free) break;
            __builtin_amdgcn_s_sleep(1);
        }
        if (!free) {
            if (lane == 0) a.out[pair * O_WORDS + O_PRODUCER_TIMEOUT] = 1;
            return;
        }
#pragma unroll
        for (int r = 0; r < kLitmusRanks; ++r) {
            V16 v;
#pragma unroll
            for (int w = 0; w < 4; ++w) v.w[w] = raw[r].w[w] + value_of(g, r, lane, w);
            st16_buffer(slot_of(a, pair, p, r, 0), lane_bytes(lane), v);
        }
        if (local) {
            // the loads stay after the stores (the wait below counts on it)
            __atomic_signal_fence(__ATOMIC_SEQ_CST);
#pragma unroll
            for (int r = 0; r < kLitmusRanks; ++r)
                raw[r] = ld16_buffer<0>(src + r * kWaveLanes * 4, lane_bytes(lane));
            // at most the 8 source loads outstanding: the slot stores have
            // reached the L2
            __builtin_amdgcn_s_waitcnt(kWaitVm | kLitmusRanks);
            __atomic_signal_fence(__ATOMIC_SEQ_CST);
        } else {
#pragma unroll
            for (int r = 0; r < kLitmusRanks; ++r)
                raw[r] = ld16_buffer<0>(src + r * kWaveLanes * 4, lane_bytes(lane));
            publish_slot(false);
        }
        if (lane < kLitmusRanks) st_flag(a.stamps + pc * kLitmusRanks + lane, g, local);
        if (lane == 0) st_flag(a.produced + pc, g, local);
    }
}

__device__ void producer(const LitmusArgs &a, int pair, int lane) {
    publish_place(a.place + pair, 0, lane);
    const bool local = partner_is_local(a.place + a.pairs + pair, 0, lane);
    if (a.prefetch) {
        producer_prefetch(a, pair, lane, local);
        return;
    }
    for (int i = 1; i <= a.trials; ++i) {
        const uint32_t g = static_cast<uint32_t>(i), p = g & 1u;
        const size_t pc = static_cast<size_t>(p) * a.pairs + pair;
        bool free = false;
        for (uint32_t spins = 0; spins < kSpins; ++spins) {
            free = ld_relaxed(a.consumed + pc) == ld_relaxed(a.produced + pc);
            if (free) break;
            __builtin_amdgcn_s_sleep(1);
        }
        if (!free) {
            if (lane == 0) a.out[pair * O_WORDS + O_PRODUCER_TIMEOUT] = 1;
            return;
        }
#pragma unroll
        for (int r = 0; r < kLitmusRanks; ++r) {
            V16 v;
#pragma unroll
            for (int w = 0; w < 4; ++w) v.w[w] = value_of(g, r, lane, w);
            *reinterpret_cast<V16 *>(slot_of(a, pair, p, r, lane)) = v;
        }
        publish_slot(local);
        if (lane < kLitmusRanks) st_flag(a.stamps + pc * kLitmusRanks + lane, g, local);
        if (lane == 0) st_flag(a.produced + pc, g, local);
    }
}

__device__ __forceinline__ void load_slot(const LitmusArgs &a, int pair, uint32_t p, int lane,
                                          V16 (&v)[kLitmusRanks]) {
#pragma unroll
    for (int r = 0; r < kLitmusRanks; ++r)
        v[r] = ld16_agent(slot_of(a, pair, p, r, 0), static_cast<uint32_t>(lane) * 16u);
}

__device__ void consumer(const LitmusArgs &a, int pair, int lane) {
    publish_place(a.place + a.pairs + pair, 0, lane);
    const uint32_t me = xcc_id();
    const bool local = partner_is_local(a.place + pair, 0, lane);
    uint32_t done = 0, bad = 0, bad_early = 0, timeouts = 0, bad_g = 0, bad_found = 0, bad_want = 0;
    const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
    for (int i = 1; i <= a.trials; ++i) {
        const uint32_t g = static_cast<uint32_t>(i), p = g & 1u;
        const size_t pc = static_cast<size_t>(p) * a.pairs + pair;
        const uint32_t *stamp = a.stamps + pc * kLitmusRanks + lane;
        V16 v[kLitmusRanks];
        bool fresh = false;
        if (a.read_first) {
            for (uint32_t spins = 0; spins < kSpins; ++spins) {
                load_slot(a, pair, p, lane, v);
                const uint32_t st = lane < kLitmusRanks ? ld_relaxed(stamp) : g;
                fresh = __ballot(st != g) == 0;
                if (fresh) break;
                __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
                __builtin_amdgcn_s_sleep(1);
            }
        } else {
            for (uint32_t spins = 0; spins < kSpins; ++spins) {
                const uint32_t st = lane < kLitmusRanks ? ld_relaxed(stamp) : g;
                fresh = __ballot(st != g) == 0;
                if (fresh) break;
                __builtin_amdgcn_s_sleep(1);
            }
            if (fresh) {
                acquire_slot(local);
                load_slot(a, pair, p, lane, v);
            }
        }
        if (!fresh) {
            timeouts = 1;
            break;
        }
        // every load of the slot has returned before it is handed back
#pragma unroll
        for (int r = 0; r < kLitmusRanks; ++r) complete(v[r]);
        if (lane == 0) st_flag(a.consumed + pc, g, local);
        // branch-free test first (it stays off the handoff's critical path);
        // the first wrong word is looked up only when there is one
        uint32_t diff = 0;
#pragma unroll
        for (int r = 0; r < kLitmusRanks; ++r)
#pragma unroll
            for (int w = 0; w < 4; ++w) diff |= v[r].w[w] ^ value_of(g, r, lane, w);
        const bool wrong = diff != 0;
        const uint64_t m = __ballot(wrong);
        ++done;
        if (m != 0) {
            if (bad == 0) {
                uint32_t found = 0, want = 0;
                bool hit = false;
#pragma unroll
                for (int r = 0; r < kLitmusRanks; ++r)
#pragma unroll
                    for (int w = 0; w < 4; ++w) {
                        const uint32_t e = value_of(g, r, lane, w);
                        const bool first = !hit && v[r].w[w] != e;
                        found = first ? v[r].w[w] : found;
                        want = first ? e : want;
                        hit = hit || first;
                    }
                const int src = __builtin_ctzll(m);
                bad_g = g;
                bad_found = __shfl(found, src);
                bad_want = __shfl(want, src);
            }
            ++bad;
            if (g <= 2) ++bad_early;
        }
    }
    const uint64_t t1 = __builtin_amdgcn_s_memrealtime();
    if (lane == 0) {
        const uint64_t peer = __hip_atomic_load(a.place + pair, __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT);
        uint32_t *o = a.out + pair * O_WORDS;
        o[O_TRIALS] = done;
        o[O_BAD] = bad;
        o[O_BAD_EARLY] = bad_early;
        o[O_TIMEOUT] = timeouts;
        o[O_PLACED] = local != static_cast<bool>(a.cross) ? 1u : 0u;
        o[O_BAD_G] = bad_g;
        o[O_BAD_FOUND] = bad_found;
        o[O_BAD_WANT] = bad_want;
        o[O_XCC] = (static_cast<uint32_t>(peer & 0xFFu) << 8) | me;
        a.ticks[pair * 2] = t0;
        a.ticks[pair * 2 + 1] = t1;
    }
}

// Grid 16 * pairs / 8 one-wave workgroups, in groups of 16: workgroups 0-7 of
// a group produce for pairs 8q + 0..7, workgroups 8-15 consume; the consumer
// of producer i is workgroup 8 + (i + shift) mod 8 (shift 1: the next XCD,
// shift 0: the same XCD).
__global__ void __launch_bounds__(kWaveLanes) litmus_kernel(LitmusArgs a) {
    const int lane = threadIdx.x;
    const int q = blockIdx.x / 16, i = blockIdx.x % 16;
    const int shift = a.cross ? 1 : 0;
    if (i < 8) {
        producer(a, 8 * q + i, lane);
    } else {
        consumer(a, 8 * q + ((i - 8 - shift + 8) & 7), lane);
    }
}

struct Buffer {
    void *p = nullptr;
    ~Buffer() {
        if (p) (void)hipFree(p);
    }
};

int hip_rc(hipError_t e) { return e == hipSuccess ? SIFAR_OK : SIFAR_EHIP; }

}  // namespace
}  // namespace sifar

extern "C" int sifar_litmus(int32_t protocol, int32_t placement, int32_t pairs, int32_t trials,
                            void *stream, sifar_litmus_result *result) {
    using namespace sifar;
    if (!result) return SIFAR_EINVAL;
    if (protocol != SIFAR_LITMUS_ORDERED && protocol != SIFAR_LITMUS_READ_FIRST &&
        protocol != SIFAR_LITMUS_ORDERED_PREFETCH)
        return SIFAR_EINVAL;
    if (placement != SIFAR_LITMUS_CROSS_XCD && placement != SIFAR_LITMUS_SAME_XCD) return SIFAR_EINVAL;
    if (pairs < 8 || pairs > kMaxPairs || pairs % 8 != 0) return SIFAR_EINVAL;
    if (trials < 1 || trials > kMaxTrials) return SIFAR_EINVAL;
    *result = sifar_litmus_result{};
    hipStream_t s = static_cast<hipStream_t>(stream);
    int dev = 0, khz = 0;
    int rc = hip_rc(hipGetDevice(&dev));
    if (!rc) rc = hip_rc(hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev));
    if (!rc && khz <= 0) rc = SIFAR_EHIP;
    if (rc) return rc;

    const size_t slot_bytes = static_cast<size_t>(pairs) * 2 * kSlotWords * sizeof(uint32_t);
    const size_t ctl_words = static_cast<size_t>(pairs) * (2 * kLitmusRanks + 2 + 2) +
                             static_cast<size_t>(pairs) * O_WORDS;
    const size_t ctl_bytes = ctl_words * sizeof(uint32_t) +
                             static_cast<size_t>(pairs) * 4 * sizeof(uint64_t);
    const size_t src_bytes = static_cast<size_t>(pairs) * kSlotWords * sizeof(uint32_t);
    Buffer slots, ctl, src;
    if (hipMalloc(&slots.p, slot_bytes) != hipSuccess) return SIFAR_ENOMEM;
    if (hipMalloc(&ctl.p, ctl_bytes) != hipSuccess) return SIFAR_ENOMEM;
    if (hipMalloc(&src.p, src_bytes) != hipSuccess) return SIFAR_ENOMEM;
    rc = hip_rc(hipMemsetAsync(slots.p, 0, slot_bytes, s));
    if (!rc) rc = hip_rc(hipMemsetAsync(ctl.p, 0, ctl_bytes, s));
    if (!rc) rc = hip_rc(hipMemsetAsync(src.p, 0, src_bytes, s));
    if (rc) return rc;

    LitmusArgs a{};
    a.slots = static_cast<uint32_t *>(slots.p);
    uint64_t *words64 = static_cast<uint64_t *>(ctl.p);
    a.place = words64;                       // 2 * pairs
    a.ticks = words64 + 2 * pairs;           // 2 * pairs
    uint32_t *w = reinterpret_cast<uint32_t *>(words64 + 4 * pairs);
    a.stamps = w;
    a.consumed = a.stamps + static_cast<size_t>(2) * pairs * kLitmusRanks;
    a.produced = a.consumed + 2 * pairs;
    a.out = a.produced + 2 * pairs;
    a.pairs = pairs;
    a.trials = trials;
    a.read_first = protocol == SIFAR_LITMUS_READ_FIRST;
    a.prefetch = protocol == SIFAR_LITMUS_ORDERED_PREFETCH;
    a.src = static_cast<const uint32_t *>(src.p);
    a.cross = placement == SIFAR_LITMUS_CROSS_XCD;
    hipLaunchKernelGGL(litmus_kernel, dim3(2 * pairs), dim3(kWaveLanes), 0, s, a);
    rc = hip_rc(hipGetLastError());
    if (rc) return rc;

    uint32_t out[kMaxPairs * O_WORDS];
    uint64_t ticks[kMaxPairs * 2];
    rc = hip_rc(hipMemcpyAsync(out, a.out, static_cast<size_t>(pairs) * O_WORDS * sizeof(uint32_t),
                               hipMemcpyDeviceToHost, s));
    if (!rc)
        rc = hip_rc(hipMemcpyAsync(ticks, a.ticks, static_cast<size_t>(pairs) * 2 * sizeof(uint64_t),
                                   hipMemcpyDeviceToHost, s));
    if (!rc) rc = hip_rc(hipStreamSynchronize(s));
    if (rc) return rc;

    double tick_sum = 0.0;
    for (int j = 0; j < pairs; ++j) {
        const uint32_t *o = out + j * O_WORDS;
        result->trials += o[O_TRIALS];
        result->violations += o[O_BAD];
        result->violations_first_epochs += o[O_BAD_EARLY];
        result->timeouts += o[O_TIMEOUT] + o[O_PRODUCER_TIMEOUT];
        result->pairs_placed += o[O_PLACED];
        if (o[O_BAD] != 0 && result->first_bad[0] == 0) {
            result->first_bad[0] = o[O_BAD_G];
            result->first_bad[1] = o[O_BAD_FOUND];
            result->first_bad[2] = o[O_BAD_WANT];
            result->first_bad[3] = o[O_XCC];
        }
        if (o[O_TRIALS] > 0) tick_sum += static_cast<double>(ticks[2 * j + 1] - ticks[2 * j]) / o[O_TRIALS];
    }
    result->pairs = static_cast<uint32_t>(pairs);
    result->ns_per_trial = tick_sum / pairs * 1e6 / static_cast<double>(khz);
    return result->timeouts != 0 ? SIFAR_EDEVICE : SIFAR_OK;
}
