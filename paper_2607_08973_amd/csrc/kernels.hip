// gfx950 (MI355X) kernels of the emulated SiFAR one-shot all-reduce.
//
// Work decomposition: a "chunk" is 512 consecutive bf16 elements of one
// token's row, handled by one 64-lane wave with one 16-byte load per rank per
// lane. Every chunk carries its own N epoch stamps (the paper's per-threadblock
// validation buffer, Sec. 4.2), so chunks validate and retry independently and
// no wave ever waits for another during the reduction proper.
//
// Memory-model choices (LLVM AMDGPU memory model for GFX942/950):
//  - stamps are read with agent-scope atomic loads (coherent across the XCDs'
//    separate L2s); the producer stores them after its payload stores, and the
//    end of the producing launch publishes both device-wide;
//  - SPEC issues the payload loads and the stamp loads together, with no
//    ordering between them (the paper's concurrent payload warps and
//    validation warp); ORDERED acquires the stamps before loading the payload;
//  - a retry starts with an acquire fence so the reloads cannot be served
//    from a stale cache line (the paper's L1-bypassing re-read, Sec. 4.2).
//
// Arithmetic: fp32 adds in ascending rank order (no reassociation, no FMA
// contraction), bf16 rounding by the native V_CVT_PK_BF16_F32 (round to nearest
// even, fp32 denormals enabled).
#include "sifar_kernels.h"

namespace sifar {
namespace {

struct alignas(16) V16 {
    uint32_t w[4];
};

__device__ __forceinline__ V16 ld16(const uint16_t *p) {
    return *reinterpret_cast<const V16 *>(p);
}

__device__ __forceinline__ void st16(uint16_t *p, const V16 &v) {
    *reinterpret_cast<V16 *>(p) = v;
}

__device__ __forceinline__ float lo_f32(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_f32(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
    const __bf16 a = static_cast<__bf16>(lo);
    const __bf16 b = static_cast<__bf16>(hi);
    return static_cast<uint32_t>(__builtin_bit_cast(uint16_t, a)) |
           (static_cast<uint32_t>(__builtin_bit_cast(uint16_t, b)) << 16);
}

__device__ __forceinline__ uint32_t ld_relaxed(const uint32_t *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ uint32_t ld_acquire(const uint32_t *p) {
    return __hip_atomic_load(p, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void st_release(uint32_t *p, uint32_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ uint32_t epoch_of(const EpochRef &e) { return e.base[0] + e.off; }

// First error wins; kind 0 means "no error".
__device__ void latch(uint32_t *err, uint32_t kind, uint32_t g, uint32_t c, uint32_t n) {
    uint32_t expected = 0;
    if (__hip_atomic_compare_exchange_strong(err, &expected, kind, __ATOMIC_RELAXED,
                                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
        __hip_atomic_store(err + 1, g, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(err + 2, c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(err + 3, n, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

constexpr uint32_t kErrRetryBudget = 1, kErrWaw = 2, kErrExchange = 3;

// ---------------------------------------------------------------------------
// Producer: the emulated peers. The wave of chunk c copies every rank's part of
// the chunk into that rank's slot of parity g & 1, then stores the N stamps
// stamp[p][c][r] = g (the peers' "write the result, then the flag" of
// Sec. 4.1). The stamp stores are ordered after the payload stores of the wave
// (workgroup-scope release). Device-wide visibility comes from the end of the
// launch: the reduction of an epoch always runs in a later launch than its
// producer (eagerly, in a step graph, and in the fused plane, which writes the
// epoch after the one its launch reduces), and the end-of-kernel release makes
// every store of a launch visible to all XCDs before the next launch starts --
// as in the paper, where the flag follows the preceding kernel's completion.
// An agent-scope release fence here would write back the XCD's whole L2 once
// per wave; measured on MI355X it costs ~0.1-0.2 us of XCD-serialised time per
// fence and caps the 38 MB all-reduce at 0.9 TB/s instead of 5.7 TB/s.
// Workgroups are numbered chunk-fastest then token, the order the reduction
// numbers its chunks, so with one wave per group the producer and the
// reduction of a chunk run on the same XCD.
template <int N>
__device__ __forceinline__ void produce_chunk(const ProduceArgs &a) {
    const int lane = threadIdx.x & (kLanes - 1);
    const Geometry &geo = a.geo;
    const int s = blockIdx.x * (blockDim.x / kLanes) + threadIdx.x / kLanes;
    if (s >= geo.segs) return;
    const int t = blockIdx.y;
    const int c = t * geo.segs + s;
    const uint32_t g = epoch_of(a.ep);
    const uint32_t p = a.ep.parity;
    const int elem_raw = s * kChunk + lane * kVec;
    const bool lane_ok = elem_raw < geo.hidden;
    const int elem = lane_ok ? elem_raw : geo.hidden - kVec;
    uint32_t *stamp = a.stamps + (static_cast<size_t>(p) * geo.w_max + c) * N;

    const uint32_t e = (g - 1u) % static_cast<uint32_t>(a.entries);
    const uint16_t *src = a.src + e * a.entry_stride + static_cast<int64_t>(t) * geo.hidden + elem;
    uint16_t *dst = a.slots + static_cast<uint64_t>(p) * geo.slot_elems +
                    static_cast<uint64_t>(t) * geo.hidden + elem;
    V16 v[N];
#pragma unroll
    for (int r = 0; r < N; ++r) v[r] = ld16(src + r * a.rank_stride);
    // Dual-buffer rule: each slot's previous epoch must have been consumed.
    const int rl = lane < N ? lane : N - 1;
    const uint32_t prev = ld_relaxed(stamp + rl);
    const uint32_t done = ld_relaxed(a.consumed + static_cast<size_t>(p) * geo.w_max + c);
    if (lane_ok) {
#pragma unroll
        for (int r = 0; r < N; ++r) st16(dst + r * 2 * geo.slot_elems, v[r]);
    }
    const uint64_t bad = __ballot(lane < N && prev != done);
    if (bad && lane == __builtin_ctzll(bad)) latch(a.err, kErrWaw, g, c, prev);

    uint32_t skip = 0;
    if (a.inject) skip = a.inject[(g - 1u) % static_cast<uint32_t>(a.inject_entries)];
    skip = (skip | (skip >> 8)) & 0xFFu;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    if (lane < N && !((skip >> lane) & 1u))
        __hip_atomic_store(stamp + lane, g, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <int N>
__global__ __launch_bounds__(1024) void produce_kernel(ProduceArgs a) {
    produce_chunk<N>(a);
}

// ---------------------------------------------------------------------------
// Reduction of one chunk per wave: speculative or ordered loads, per-rank
// stamp validation by ballot, bounded retry, fp32 sum in rank order, bf16
// store. With EPI the fused residual-add + RMSNorm follows; the token's sum of
// squares is combined across the waves of the workgroup (LDS) and across the
// workgroups of the token (epoch-tagged exchange words).
// FUSED: the grid has a second plane (blockIdx.z == 1) of producer workgroups
// that write the NEXT epoch (other parity) while the first plane reduces this
// one -- the emulated peers running one epoch ahead, which is as far ahead as
// two slots allow. The planes touch disjoint slots and stamps.
template <int N, int MODE, bool EPI, bool FUSED>
__global__ __launch_bounds__(1024) void reduce_kernel(ReduceArgs a, ProduceArgs pa) {
    if (FUSED && blockIdx.z == 1) {
        produce_chunk<N>(pa);
        return;
    }
    const int lane = threadIdx.x & (kLanes - 1);
    const int wave = threadIdx.x / kLanes;
    const int G = blockDim.x / kLanes;
    const Geometry &geo = a.geo;

    // grid: x = chunk groups of a token, y = token
    const int t = blockIdx.y;
    const int s = blockIdx.x * G + wave;
    if (!EPI && s >= geo.segs) return;
    // EPI: trailing waves of a token's last group idle but join the barriers;
    // every lane loads in bounds (clamped) and only lane_ok lanes store.
    const bool active = s < geo.segs;
    const int sc = active ? s : geo.segs - 1;
    const int c = t * geo.segs + sc;
    const int elem_raw = s * kChunk + lane * kVec;
    const bool lane_ok = active && elem_raw < geo.hidden;
    const int elem = sc * kChunk + lane * kVec < geo.hidden ? sc * kChunk + lane * kVec
                                                            : geo.hidden - kVec;
    const uint32_t p = a.ep.parity;
    const uint64_t row = static_cast<uint64_t>(t) * geo.hidden + elem;

    const uint16_t *slot0 = a.slots + static_cast<uint64_t>(p) * geo.slot_elems + row;
    const uint64_t rank_step = 2 * geo.slot_elems;  // slots are [rank][parity]
    uint32_t *stamp = a.stamps + (static_cast<size_t>(p) * geo.w_max + c) * N;

    V16 v[N];
    V16 rv, wv;
    if (EPI) {
        rv = ld16(a.residual + row);
        wv = ld16(a.weight + elem);
    }
    const uint32_t g = epoch_of(a.ep);

    uint32_t st = 0;
    if (MODE == kOrdered) {
        if (active && lane < N) st = ld_acquire(stamp + lane);
    } else {
#pragma unroll
        for (int r = 0; r < N; ++r) v[r] = ld16(slot0 + r * rank_step);
        if (MODE == kSpec && active && lane < N) st = ld_relaxed(stamp + lane);
    }

    uint32_t attempts = 1, first = 0, last = 0;
    if (MODE != kNone && active) {
        uint32_t m = static_cast<uint32_t>(__ballot(lane < N && st != g));
        first = last = m;
        bool fail = m != 0 || a.forced_retries >= 1;
        while (fail) {
            if (attempts >= a.max_attempts) {
                if (lane == 0) latch(a.err, kErrRetryBudget, g, c, attempts);
                break;
            }
            if (attempts == 1 && a.inject && m != 0) {
                // Deterministic injection: the late ranks catch up right now.
                const uint32_t inj = a.inject[(g - 1u) % static_cast<uint32_t>(a.inject_entries)];
                if (lane < N && ((inj >> lane) & 1u) && !((inj >> (8 + lane)) & 1u))
                    st_release(stamp + lane, g);
            }
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
            if (MODE == kOrdered) {
                if (lane < N) st = ld_acquire(stamp + lane);
            } else {
                if (lane < N) st = ld_relaxed(stamp + lane);
#pragma unroll
                for (int r = 0; r < N; ++r) v[r] = ld16(slot0 + r * rank_step);
            }
            ++attempts;
            m = static_cast<uint32_t>(__ballot(lane < N && st != g));
            last = m;
            fail = m != 0 || attempts <= a.forced_retries;
        }
    }
    if (MODE == kOrdered) {
#pragma unroll
        for (int r = 0; r < N; ++r) v[r] = ld16(slot0 + r * rank_step);
    }

    // Fixed-order fp32 sum: acc = x_0; acc += x_1; ... acc += x_{N-1}.
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

    if (active && lane == 0) {
        const uint32_t word = (attempts > 0xFFFFu ? 0xFFFFu : attempts) | ((first & 0xFFu) << 16) |
                              ((last & 0xFFu) << 24);
        a.log[static_cast<size_t>((g - 1u) % static_cast<uint32_t>(a.log_epochs)) * geo.w_max + c] =
            word;
        a.consumed[static_cast<size_t>(p) * geo.w_max + c] = g;
    }

    if (!EPI) {
        if (lane_ok) st16(a.out + row, o);
        return;
    }

    // ---- fused residual-add + RMSNorm -------------------------------------
    // res' = bf16(a + res), with a = the bf16 all-reduce result.
    V16 nr;
    float x[kVec];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const float a0 = lo_f32(o.w[k]), a1 = hi_f32(o.w[k]);
        nr.w[k] = pack_bf16(a0 + lo_f32(rv.w[k]), a1 + hi_f32(rv.w[k]));
        x[2 * k] = lo_f32(nr.w[k]);
        x[2 * k + 1] = hi_f32(nr.w[k]);
    }
    if (lane_ok) st16(a.residual + row, nr);

    float ss = 0.f;
    if (lane_ok) {
#pragma unroll
        for (int k = 0; k < kVec; ++k) ss = __builtin_fmaf(x[k], x[k], ss);
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
            const int q = blockIdx.x;
            uint64_t *ex = a.exch + static_cast<size_t>(t) * Q;
            if (lane == 0) {
                const uint64_t word = (static_cast<uint64_t>(g) << 32) | __float_as_uint(grp);
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
            if (!ready && lane == 0) latch(a.err, kErrExchange, g, c, spins);
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
    for (int k = 0; k < 4; ++k) {
        const float w0 = lo_f32(wv.w[k]), w1 = hi_f32(wv.w[k]);
        yo.w[k] = pack_bf16((x[2 * k] * inv) * w0, (x[2 * k + 1] * inv) * w1);
    }
    if (lane_ok) st16(a.y + row, yo);
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
    if (pa) {
        grid.z = 2;
        if (epi)
            hipLaunchKernelGGL((reduce_kernel<N, MODE, true, true>), grid, block, 0, s, a, *pa);
        else
            hipLaunchKernelGGL((reduce_kernel<N, MODE, false, true>), grid, block, 0, s, a, *pa);
    } else {
        if (epi)
            hipLaunchKernelGGL((reduce_kernel<N, MODE, true, false>), grid, block, 0, s, a, none);
        else
            hipLaunchKernelGGL((reduce_kernel<N, MODE, false, false>), grid, block, 0, s, a, none);
    }
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

int max_active_groups(int nranks, int mode, bool epilogue, int waves_per_group) {
    const void *fn = nullptr;
#define SIFAR_PICK(NN)                                                                  \
    if (nranks == NN) {                                                                 \
        if (mode == kSpec)                                                              \
            fn = epilogue ? (const void *)reduce_kernel<NN, kSpec, true, true>          \
                          : (const void *)reduce_kernel<NN, kSpec, false, false>;       \
        else if (mode == kOrdered)                                                      \
            fn = epilogue ? (const void *)reduce_kernel<NN, kOrdered, true, true>       \
                          : (const void *)reduce_kernel<NN, kOrdered, false, false>;    \
        else                                                                            \
            fn = epilogue ? (const void *)reduce_kernel<NN, kNone, true, true>          \
                          : (const void *)reduce_kernel<NN, kNone, false, false>;       \
    }
    SIFAR_PICK(1) SIFAR_PICK(2) SIFAR_PICK(3) SIFAR_PICK(4)
    SIFAR_PICK(5) SIFAR_PICK(6) SIFAR_PICK(7) SIFAR_PICK(8)
#undef SIFAR_PICK
    if (!fn) return 0;
    int per_cu = 0, dev = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, waves_per_group * kLanes, 0) !=
        hipSuccess)
        return 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return 0;
    return per_cu * cus;
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
