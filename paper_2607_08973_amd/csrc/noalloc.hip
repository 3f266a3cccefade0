// Allocation-free all-reduce: one epoch of the emulated one-shot all-reduce
// (the peers' write, then the speculative reduction, Sec. 3.5 and 4.2) with
// every piece of library state -- slots, stamps, consumed/produced words, the
// decision log, the epoch base and the error word -- in one static device
// array, for callers that cannot allocate device memory. It runs the same
// producer and reduction kernels as sifar_produce + sifar_reduce.
//
// The array's name is a host-side stand-in in host code, not a device
// address: each GPU holds its own copy at its own address, which
// hipGetSymbolAddress returns once per device (with that device current) at
// the first call there. Only that address is handed to kernels.
#include <hip/hip_runtime.h>

#include <mutex>

#include "sifar.h"
#include "sifar_kernels.h"

namespace sifar {
namespace {

constexpr int kMaxDevices = 64;
constexpr uint64_t kSlotElems = SIFAR_NOALLOC_MAX_ELEMS;   // elements between two slots
constexpr int kWMax = SIFAR_NOALLOC_MAX_TOKENS + SIFAR_NOALLOC_MAX_ELEMS / kChunk;  // chunk bound
constexpr uint32_t kAttempts = 1024;  // retry budget (validation cannot fail without an overlap)

// Byte offsets inside the array, each on a 256-byte boundary.
constexpr uint64_t align256(uint64_t b) { return (b + 255) / 256 * 256; }
constexpr uint64_t kOffState = 0;
constexpr uint64_t kOffStamps = align256(kOffState + sizeof(DevState));
constexpr uint64_t kOffConsumed = align256(kOffStamps + 2ull * kWMax * kMaxRanks * 4);
constexpr uint64_t kOffProduced = align256(kOffConsumed + 2ull * kWMax * 4);
constexpr uint64_t kOffLog = align256(kOffProduced + 2ull * kWMax * 4);
constexpr uint64_t kOffSlots = align256(kOffLog + 1ull * kWMax * 4);
constexpr uint64_t kScratchBytes = kOffSlots + 2ull * kMaxRanks * 2 * kSlotElems;
static_assert(kScratchBytes <= SIFAR_NOALLOC_SCRATCH_BYTES, "header states the array's size");

// Zero at load time, so every stamp starts stale and every chunk's consumed
// and produced words agree (its slots are free).
static __device__ __align__(256) unsigned char scratch[SIFAR_NOALLOC_SCRATCH_BYTES];

struct PerDevice {
    unsigned char *ptr = nullptr;  // this device's copy of `scratch`
    uint32_t next_epoch = 1;       // epochs of earlier calls on this device are smaller
};

std::mutex g_mutex;
PerDevice g_dev[kMaxDevices];

}  // namespace
}  // namespace sifar

extern "C" int sifar_allreduce_noalloc(const void *src, int64_t src_rank_stride, int32_t nranks,
                                       int32_t tokens, int32_t hidden, void *out, void *stream) {
    using namespace sifar;
    if (!src || !out || (reinterpret_cast<uintptr_t>(src) & 15u) ||
        (reinterpret_cast<uintptr_t>(out) & 15u))
        return SIFAR_EINVAL;
    if (nranks < 1 || nranks > kMaxRanks) return SIFAR_EINVAL;
    if (hidden < 8 || hidden > 65536 || hidden % 8) return SIFAR_EINVAL;
    if (tokens < 1 || tokens > SIFAR_NOALLOC_MAX_TOKENS) return SIFAR_EINVAL;
    if (static_cast<int64_t>(tokens) * hidden > SIFAR_NOALLOC_MAX_ELEMS) return SIFAR_EINVAL;
    if (src_rank_stride % 8 || src_rank_stride < static_cast<int64_t>(tokens) * hidden)
        return SIFAR_EINVAL;
    if (tokens * ((hidden + kChunk - 1) / kChunk) > kWMax) return SIFAR_EINVAL;  // never, by the above
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return SIFAR_EHIP;
    if (dev < 0 || dev >= kMaxDevices) return SIFAR_EINVAL;

    unsigned char *base = nullptr;
    uint32_t g = 0;
    {
        std::lock_guard<std::mutex> lock(g_mutex);
        PerDevice &d = g_dev[dev];
        if (!d.ptr) {
            void *p = nullptr;
            if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return SIFAR_EHIP;
            d.ptr = static_cast<unsigned char *>(p);
        }
        base = d.ptr;
        g = d.next_epoch;
        d.next_epoch = g + 1u == 0u ? 1u : g + 1u;  // epoch 0 would equal a never-written stamp
    }

    DevState *state = reinterpret_cast<DevState *>(base + kOffState);
    Geometry geo{};
    geo.nranks = nranks;
    geo.tokens = tokens;
    geo.hidden = hidden;
    geo.segs = (hidden + kChunk - 1) / kChunk;
    geo.w_max = kWMax;
    geo.slot_elems = kSlotElems;
    // the epoch is passed whole: base = the always-zero word
    const EpochRef ep{&state->zero, g, g & 1u};

    ProduceArgs pa{};
    pa.geo = geo;
    pa.ep = ep;
    pa.slots = reinterpret_cast<uint16_t *>(base + kOffSlots);
    pa.stamps = reinterpret_cast<uint32_t *>(base + kOffStamps);
    pa.consumed = reinterpret_cast<const uint32_t *>(base + kOffConsumed);
    pa.produced = reinterpret_cast<uint32_t *>(base + kOffProduced);
    pa.src = static_cast<const uint16_t *>(src);
    pa.entry_stride = 0;
    pa.rank_stride = src_rank_stride;
    pa.entries = 1;
    pa.entries_div = make_div(1);
    pa.inject_div = make_div(1);
    pa.err = state->err;

    ReduceArgs ra{};
    ra.geo = geo;
    ra.ep = ep;
    ra.slots = pa.slots;
    ra.stamps = pa.stamps;
    ra.consumed = reinterpret_cast<uint32_t *>(base + kOffConsumed);
    ra.log = reinterpret_cast<uint32_t *>(base + kOffLog);
    ra.log_epochs = 1;
    ra.log_div = make_div(1);
    ra.inject_div = make_div(1);
    ra.max_attempts = kAttempts;
    ra.spin_limit = 1;
    ra.out = static_cast<uint16_t *>(out);
    ra.groups_per_token = 1;
    ra.err = state->err;

    hipStream_t s = static_cast<hipStream_t>(stream);
    if (launch_produce(pa, 1, s) != hipSuccess) return SIFAR_EHIP;
    if (launch_reduce(ra, nullptr, kSpec, false, 1, s) != hipSuccess) return SIFAR_EHIP;
    return SIFAR_OK;
}
