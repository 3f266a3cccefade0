// Internal interface between the host runtime (api.cpp) and the gfx950
// kernels (kernels.hip). Not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sifar {

constexpr int kLanes = 64;                 // wavefront width on CDNA
constexpr int kVec = 8;                    // bf16 elements per 16-byte load
constexpr int kChunk = kLanes * kVec;      // elements per chunk: one wave, one load per rank per lane
constexpr int kMaxRanks = 8;
constexpr int kMaxWavesPerGroup = 16;
constexpr int kChainGroupWaves = 4;         // waves per persistent-step workgroup when grouped
constexpr int kExchPlanes = 4;              // epoch-indexed planes of the epilogue exchange

// x % d for a divisor fixed per launch, by a multiply-high instead of a
// division sequence (Granlund and Montgomery, "Division by invariant integers
// using multiplication", 1994, unsigned case): with l = ceil(log2 d) and
// m = floor(2^32 (2^l - d) / d) + 1, the quotient of a 32-bit x is
// (t + ((x - t) >> min(l, 1))) >> max(l - 1, 0), t = the high word of m * x.
struct DivU32 {
    uint32_t m, sh1, sh2, d;
};

__host__ __device__ inline DivU32 make_div(uint32_t d) {
    uint32_t l = 0;
    while (l < 32 && (uint64_t{1} << l) < d) ++l;
    DivU32 v;
    v.m = static_cast<uint32_t>(((uint64_t{1} << 32) * ((uint64_t{1} << l) - d)) / d + 1);
    v.sh1 = l < 1 ? l : 1;
    v.sh2 = l > 1 ? l - 1 : 0;
    v.d = d;
    return v;
}

__host__ __device__ inline uint32_t mod_u32(uint32_t x, const DivU32 &v) {
    const uint32_t t = static_cast<uint32_t>((static_cast<uint64_t>(v.m) * x) >> 32);
    const uint32_t q = (t + ((x - t) >> v.sh1)) >> v.sh2;
    return x - q * v.d;
}

// Device-resident state shared by all kernels of a handle.
struct DevState {
    uint32_t epoch_base;   // graph nodes compute g = epoch_base + node offset
    uint32_t zero;         // always 0: eager launches pass g as the offset
    uint32_t err[4];       // kind, epoch, chunk, attempts (first error wins)
    uint32_t chain_done;   // waves of the running persistent step that have finished
};

// Geometry common to the producer and the reduction.
struct Geometry {
    int32_t nranks;
    int32_t tokens;
    int32_t hidden;
    int32_t segs;          // chunks per token = ceil(hidden / kChunk)
    int32_t w_max;         // max_tokens * segs: stride of the stamp and log rows
    uint64_t slot_elems;   // elements between consecutive slots
};

// Where the epoch of a launch comes from: g = *base + off. The slot parity is
// frozen at launch (graph capture) time -- g & 1 with dual buffering (the host
// keeps *base even for graphs), 0 with a single buffer.
struct EpochRef {
    const uint32_t *base;
    uint32_t off;
    uint32_t parity;
};

struct ProduceArgs {
    Geometry geo;
    EpochRef ep;
    uint16_t *slots;             // [N][2][slot_elems]
    uint32_t *stamps;            // [2][w_max][N]
    const uint32_t *consumed;    // [2][w_max]: last epoch whose reduction finished the chunk
    uint32_t *produced;          // [2][w_max]: last epoch written into the chunk's slots
    const uint16_t *src;         // entry e, rank r: src + e*entry_stride + r*rank_stride
    int64_t entry_stride;
    int64_t rank_stride;
    int32_t entries;             // epoch g uses entry (g - 1) % entries
    DivU32 entries_div;          // make_div(entries)
    const uint16_t *inject;      // [inject_entries] late | withheld << 8, or null
    int32_t inject_entries;
    DivU32 inject_div;           // make_div(inject_entries), or make_div(1) without a table
    uint16_t *stage;             // [N][2][slot_elems], or null: with deterministic injection a
                                 // late rank's payload is written here, not into its slot, and
                                 // the reduction moves it into the slot when the rank catches up
    uint32_t *err;
};

struct ReduceArgs {
    Geometry geo;
    EpochRef ep;
    uint16_t *slots;             // written only when a late rank catches up (deterministic injection)
    uint32_t *stamps;
    uint32_t *consumed;
    uint32_t *log;               // [log_epochs][w_max]
    uint32_t *stamp_log;         // [log_epochs][w_max][2][N]: the raw stamps of the chunk's first
                                 // and last validation (per-epoch launches: may be null)
    int32_t log_epochs;
    DivU32 log_div;              // make_div(log_epochs)
    uint32_t max_attempts;
    uint32_t forced_retries;
    uint32_t spin_limit;
    const uint16_t *inject;
    int32_t inject_entries;
    DivU32 inject_div;
    const uint16_t *stage;       // late ranks' payload (ProduceArgs::stage), or null
    uint16_t *out;               // plain: [tokens][hidden]
    uint16_t *residual;          // epilogue: [tokens][hidden], in place
    const uint16_t *weight;      // [hidden]
    uint16_t *y;                 // [tokens][hidden]
    uint64_t *exch;              // [kExchPlanes][max_tokens][groups_per_token]: (epoch << 32) |
                                 // partial bits; per-launch epilogues use planes g & 1,
                                 // persistent steps g mod kExchPlanes
    int32_t groups_per_token;
    int32_t exch_parity_stride;  // max_tokens * groups_per_token
    float eps;
    uint32_t *err;
};

// One launch running a whole decode step: consumer waves (plane 0) reduce the
// L epochs one after another while producer waves (plane 1) play the peers,
// concurrently, synchronised only through stamps and consumed/produced words.
struct ChainArgs {
    ReduceArgs r;                // r.out / r.y point at ring entry 0
    ProduceArgs p;
    int32_t reduces;             // L
    uint64_t ring_stride;        // elements between ring entries
    uint32_t late_delay;         // injected late stamps land after this many sleeps
    uint32_t *epoch_base;        // advanced by `advance` by the last wave to finish
    uint32_t advance;
    uint32_t *done;              // arrival counter of the step's waves (left at 0)
    uint32_t parity_mask;        // 1: dual buffering (parity = epoch & 1); 0: one slot
    uint64_t *place;             // [2][w_max]: plane 0 consumer, plane 1 producer of each
                                 // chunk: (base + 1) << 32 | 0x100 | XCD, written at step start
};

enum Mode : int { kSpec = 0, kOrdered = 1, kNone = 2 };

hipError_t launch_produce(const ProduceArgs &a, int waves_per_group, hipStream_t s);
// With `next` non-null the launch also produces the next epoch (fused peers).
hipError_t launch_reduce(const ReduceArgs &a, const ProduceArgs *next, int mode, bool epilogue,
                         int waves_per_group, hipStream_t s);
// Workgroups of the reduction kernel that can be resident at once on the
// current device (0 if unknown).
int max_active_groups(int nranks, int mode, bool epilogue, int waves_per_group);
// Same for the persistent chain kernel's workgroups of `waves` waves (1 or
// kChainGroupWaves); `prefetch` picks the one-wave kernel whose producer loads
// an epoch's sources ahead (more registers, lower occupancy).
int max_active_chain_groups(int nranks, int mode, bool epilogue, int waves, bool prefetch);
// Persistent step: grid (segs / waves, tokens, 2); waves = 1, or
// kChainGroupWaves (segs divisible by it, waves * nranks <= 64) to let one
// release fence cover a workgroup's chunks.
hipError_t launch_chain(const ChainArgs &a, int mode, bool epilogue, int waves, bool prefetch,
                        hipStream_t s);
hipError_t launch_advance(uint32_t *epoch_base, uint32_t step, hipStream_t s);
hipError_t launch_set_base(uint32_t *epoch_base, uint32_t value, hipStream_t s);
hipError_t launch_fill_u32(uint32_t *p, uint32_t value, uint64_t count, hipStream_t s);

}  // namespace sifar
