// Latency floors of one MI355X, the yardsticks the all-reduce's latency is read
// against: what a graph node, an eager launch, an agent-scope atomic, an
// acquire load, a coherent load, a load of recently read data, a load that
// misses every cache, an agent-scope release fence and a release -> acquire
// handoff between two XCDs cost on their own.
//
// Each device-side probe is one wave whose lane 0 runs a chain of dependent
// operations (every address depends on the previous result, so the operations
// cannot overlap) between two reads of the 100 MHz real-time counter. The
// handoff probe runs two such waves in different workgroups; workgroups are
// dealt to the 8 XCDs round robin, so workgroups 0 and 1 sit on different XCDs
// and workgroups 0 and 8 on the same one (the XCC_ID register read in the
// kernel confirms where each ran). Every wait is bounded.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "sifar.h"

namespace {

constexpr uint32_t kSpinLimit = 1u << 20;  // polls per handoff before giving up
constexpr int kMaxIterations = 1 << 20;
constexpr int kMaxChase = 1 << 16;         // hops of the cache-missing chase

// result words written by the probes
enum { R_T0 = 0, R_T1 = 1, R_OK = 2, R_XCC_A = 3, R_XCC_B = 4, R_SINK = 5, R_WORDS = 8 };

__device__ __forceinline__ uint64_t now() { return __builtin_amdgcn_s_memrealtime(); }

__device__ __forceinline__ uint32_t xcc_id() {
    uint32_t v;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID, 0, 4)" : "=s"(v));
    return v;
}

__global__ void empty_kernel() {}

__global__ void __launch_bounds__(64) atomic_chain(uint32_t *w, int iters, uint64_t *res) {
    if (threadIdx.x != 0) return;
    uint32_t v = 0;
    const uint64_t t0 = now();
    for (int i = 0; i < iters; ++i)
        v = __hip_atomic_fetch_add(w + (v >> 31), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const uint64_t t1 = now();
    res[R_T0] = t0;
    res[R_T1] = t1;
    res[R_OK] = 1;
    res[R_XCC_A] = xcc_id();
    res[R_SINK] = v;
}

// w[0] == 0 throughout, so every load reads index 0, through an address that
// depends on the previous load.
template <int ORDER>
__global__ void __launch_bounds__(64) load_chain(const uint32_t *w, int iters, uint64_t *res) {
    if (threadIdx.x != 0) return;
    uint32_t v = 0;
    const uint64_t t0 = now();
    for (int i = 0; i < iters; ++i)
        v = __hip_atomic_load(w + (v >> 31), ORDER, __HIP_MEMORY_SCOPE_AGENT);
    const uint64_t t1 = now();
    res[R_T0] = t0;
    res[R_T1] = t1;
    res[R_OK] = 1;
    res[R_XCC_A] = xcc_id();
    res[R_SINK] = v;
}

// 16-byte pointer chase: entry i holds the index of the next entry.
__global__ void chase_init(uint4 *p, uint64_t n, uint64_t stride) {
    for (uint64_t i = blockIdx.x * static_cast<uint64_t>(blockDim.x) + threadIdx.x; i < n;
         i += static_cast<uint64_t>(gridDim.x) * blockDim.x)
        p[i] = make_uint4(static_cast<uint32_t>((i + stride) & (n - 1)), 0u, 0u, 0u);
}

__global__ void scrub(uint4 *p, uint64_t n) {
    for (uint64_t i = blockIdx.x * static_cast<uint64_t>(blockDim.x) + threadIdx.x; i < n;
         i += static_cast<uint64_t>(gridDim.x) * blockDim.x)
        p[i] = make_uint4(static_cast<uint32_t>(i), 1u, 2u, 3u);
}

__global__ void __launch_bounds__(64) chase(const uint4 *p, int warm, int iters, uint64_t *res) {
    if (threadIdx.x != 0) return;
    uint32_t idx = 0;
    for (int i = 0; i < warm; ++i) idx = p[idx].x;
    const uint64_t t0 = now();
    for (int i = 0; i < iters; ++i) idx = p[idx].x;
    const uint64_t t1 = now();
    res[R_T0] = t0;
    res[R_T1] = t1;
    res[R_OK] = 1;
    res[R_XCC_A] = xcc_id();
    res[R_SINK] = idx;
}

// A 16-byte store followed by an agent-scope release fence, repeated; the
// next store's address depends on a load issued after the fence.
__global__ void __launch_bounds__(64) fence_chain(uint4 *p, int iters, uint64_t *res) {
    if (threadIdx.x != 0) return;
    uint32_t v = 0;
    const uint64_t t0 = now();
    for (int i = 0; i < iters; ++i) {
        p[(i & 63) + (v >> 31)] = make_uint4(static_cast<uint32_t>(i), v, 0u, 0u);
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
        v = __hip_atomic_load(reinterpret_cast<const uint32_t *>(p + 64), __ATOMIC_RELAXED,
                              __HIP_MEMORY_SCOPE_AGENT);
    }
    const uint64_t t1 = now();
    res[R_T0] = t0;
    res[R_T1] = t1;
    res[R_OK] = 1;
    res[R_XCC_A] = xcc_id();
    res[R_SINK] = v;
}

// Workgroup 0 and workgroup `partner` hand a counter back and forth: each
// waits (relaxed agent-scope polling, then an acquire fence) for its turn's
// value and release-stores the next one. Other workgroups exit at once.
__global__ void __launch_bounds__(64) pingpong(uint32_t *flag, int iters, int partner,
                                               uint64_t *res) {
    const int wg = blockIdx.x;
    if (threadIdx.x != 0 || (wg != 0 && wg != partner)) return;
    const bool first = wg == 0;
    res[first ? R_XCC_A : R_XCC_B] = xcc_id();
    bool ok = true;
    const uint64_t t0 = now();
    for (int k = 0; k < iters && ok; ++k) {
        const uint32_t want = 2u * static_cast<uint32_t>(k) + (first ? 0u : 1u);
        uint32_t spins = 0;
        while (__hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != want) {
            if (++spins > kSpinLimit) {
                ok = false;
                break;
            }
        }
        if (!ok) break;
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        __hip_atomic_store(flag, want + 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
    }
    if (first) {
        uint32_t spins = 0;
        const uint32_t last = 2u * static_cast<uint32_t>(iters);
        while (ok && __hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != last)
            if (++spins > kSpinLimit) ok = false;
        const uint64_t t1 = now();
        res[R_T0] = t0;
        res[R_T1] = t1;
        res[R_OK] = ok ? 1 : 0;
    } else if (!ok) {
        res[R_SINK] = 1;  // the second wave gave up
    }
}

struct Scoped {
    void *p = nullptr;
    ~Scoped() {
        if (p) (void)hipFree(p);
    }
};

int alloc(Scoped &s, size_t bytes) {
    return hipMalloc(&s.p, bytes) == hipSuccess ? SIFAR_OK : SIFAR_ENOMEM;
}

int hip_ok(hipError_t e) { return e == hipSuccess ? SIFAR_OK : SIFAR_EHIP; }

int launch_ok() { return hip_ok(hipGetLastError()); }

// Host-timed floors: a hipGraph of `nodes` empty kernels, or `nodes` eager
// launches, timed with events over several repetitions.
int host_floor(int kind, int nodes, hipStream_t s, double *ns) {
    hipEvent_t e0 = nullptr, e1 = nullptr;
    hipGraph_t g = nullptr;
    hipGraphExec_t ge = nullptr;
    hipStream_t cap = nullptr;
    int rc = hip_ok(hipEventCreate(&e0));
    if (!rc) rc = hip_ok(hipEventCreate(&e1));
    constexpr int kReps = 10;
    if (!rc && kind == SIFAR_FLOOR_GRAPH_NODE) {
        rc = hip_ok(hipStreamCreateWithFlags(&cap, hipStreamNonBlocking));
        if (!rc) rc = hip_ok(hipStreamBeginCapture(cap, hipStreamCaptureModeThreadLocal));
        if (!rc) {
            for (int i = 0; i < nodes; ++i) hipLaunchKernelGGL(empty_kernel, dim3(1), dim3(64), 0, cap);
            const int lrc = launch_ok();
            const int crc = hip_ok(hipStreamEndCapture(cap, &g));
            rc = lrc ? lrc : crc;
        }
        if (!rc) rc = hip_ok(hipGraphInstantiate(&ge, g, nullptr, nullptr, 0));
        for (int w = 0; !rc && w < 2; ++w) rc = hip_ok(hipGraphLaunch(ge, s));
        if (!rc) rc = hip_ok(hipEventRecord(e0, s));
        for (int r = 0; !rc && r < kReps; ++r) rc = hip_ok(hipGraphLaunch(ge, s));
        if (!rc) rc = hip_ok(hipEventRecord(e1, s));
    } else if (!rc) {
        for (int i = 0; i < nodes; ++i) hipLaunchKernelGGL(empty_kernel, dim3(1), dim3(64), 0, s);
        rc = launch_ok();
        if (!rc) rc = hip_ok(hipEventRecord(e0, s));
        for (int r = 0; !rc && r < kReps; ++r) {
            for (int i = 0; i < nodes; ++i) hipLaunchKernelGGL(empty_kernel, dim3(1), dim3(64), 0, s);
            rc = launch_ok();
        }
        if (!rc) rc = hip_ok(hipEventRecord(e1, s));
    }
    if (!rc) rc = hip_ok(hipEventSynchronize(e1));
    float ms = 0.f;
    if (!rc) rc = hip_ok(hipEventElapsedTime(&ms, e0, e1));
    if (!rc) *ns = static_cast<double>(ms) * 1e6 / (static_cast<double>(kReps) * nodes);
    if (ge) (void)hipGraphExecDestroy(ge);
    if (g) (void)hipGraphDestroy(g);
    if (cap) (void)hipStreamDestroy(cap);
    if (e0) (void)hipEventDestroy(e0);
    if (e1) (void)hipEventDestroy(e1);
    return rc;
}

}  // namespace

extern "C" int sifar_floor(int32_t kind, int32_t iterations, void *stream, double *ns_per_op,
                           uint32_t info[4]) {
    if (!ns_per_op || !info || iterations < 1 || iterations > kMaxIterations) return SIFAR_EINVAL;
    if (kind < SIFAR_FLOOR_GRAPH_NODE || kind > SIFAR_FLOOR_PINGPONG_SAME_XCD) return SIFAR_EINVAL;
    if ((kind == SIFAR_FLOOR_COLD_LOAD || kind == SIFAR_FLOOR_PINGPONG_XCD ||
         kind == SIFAR_FLOOR_PINGPONG_SAME_XCD) && iterations > kMaxChase)
        return SIFAR_EINVAL;
    hipStream_t s = static_cast<hipStream_t>(stream);
    info[0] = info[1] = info[2] = info[3] = 0;
    *ns_per_op = 0.0;
    if (kind == SIFAR_FLOOR_GRAPH_NODE || kind == SIFAR_FLOOR_EAGER_LAUNCH) {
        if (iterations > 4096) return SIFAR_EINVAL;
        const int rc = host_floor(kind, iterations, s, ns_per_op);
        info[0] = rc == SIFAR_OK;
        return rc;
    }

    int dev = 0, khz = 0;
    int rc = hip_ok(hipGetDevice(&dev));
    if (!rc) rc = hip_ok(hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev));
    if (!rc && khz <= 0) rc = SIFAR_EHIP;
    Scoped res, words, big, dirt;
    if (!rc) rc = alloc(res, R_WORDS * sizeof(uint64_t));
    if (!rc) rc = hip_ok(hipMemsetAsync(res.p, 0, R_WORDS * sizeof(uint64_t), s));
    if (rc) return rc;
    uint64_t *r = static_cast<uint64_t *>(res.p);
    const dim3 wave(64);
    switch (kind) {
    case SIFAR_FLOOR_ATOMIC:
    case SIFAR_FLOOR_ACQUIRE_LOAD:
    case SIFAR_FLOOR_COHERENT_LOAD:
    case SIFAR_FLOOR_PINGPONG_XCD:
    case SIFAR_FLOOR_PINGPONG_SAME_XCD: {
        rc = alloc(words, 256);
        if (!rc) rc = hip_ok(hipMemsetAsync(words.p, 0, 256, s));
        uint32_t *w = static_cast<uint32_t *>(words.p);
        if (rc) break;
        if (kind == SIFAR_FLOOR_ATOMIC)
            hipLaunchKernelGGL(atomic_chain, dim3(1), wave, 0, s, w, iterations, r);
        else if (kind == SIFAR_FLOOR_ACQUIRE_LOAD)
            hipLaunchKernelGGL(load_chain<__ATOMIC_ACQUIRE>, dim3(1), wave, 0, s, w, iterations, r);
        else if (kind == SIFAR_FLOOR_COHERENT_LOAD)
            hipLaunchKernelGGL(load_chain<__ATOMIC_RELAXED>, dim3(1), wave, 0, s, w, iterations, r);
        else {
            const int partner = kind == SIFAR_FLOOR_PINGPONG_XCD ? 1 : 8;
            hipLaunchKernelGGL(pingpong, dim3(partner + 1), wave, 0, s, w, iterations, partner, r);
        }
        rc = launch_ok();
        break;
    }
    case SIFAR_FLOOR_WARM_LOAD:
    case SIFAR_FLOOR_COLD_LOAD: {
        // Warm: a 1 MiB ring (more than the CU's L1, less than the XCD's L2)
        // walked line after line, so address translation stays warm, after
        // one pass over it. Cold: a 1 GiB ring walked 4 MiB + 4224 B at a time,
        // every hop a new line and a new translation, after 512 MiB of
        // unrelated writes have pushed it out of L2 and the Infinity Cache.
        const bool cold = kind == SIFAR_FLOOR_COLD_LOAD;
        const uint64_t n = cold ? (uint64_t(1) << 26) : (uint64_t(1) << 16);  // 16-B entries
        const uint64_t stride = cold ? (262144 + 264) : 8;  // in entries
        rc = alloc(big, n * sizeof(uint4));
        if (!rc && cold) rc = alloc(dirt, size_t(512) << 20);
        if (rc) break;
        uint4 *p = static_cast<uint4 *>(big.p);
        hipLaunchKernelGGL(chase_init, dim3(1024), dim3(256), 0, s, p, n, stride);
        if (cold)
            hipLaunchKernelGGL(scrub, dim3(2048), dim3(256), 0, s, static_cast<uint4 *>(dirt.p),
                               (uint64_t(512) << 20) / sizeof(uint4));
        const int warm = cold ? 0 : static_cast<int>(n / 8);
        hipLaunchKernelGGL(chase, dim3(1), wave, 0, s, p, warm, iterations, r);
        rc = launch_ok();
        break;
    }
    case SIFAR_FLOOR_RELEASE_FENCE: {
        rc = alloc(words, 65 * sizeof(uint4));
        if (!rc) rc = hip_ok(hipMemsetAsync(words.p, 0, 65 * sizeof(uint4), s));
        if (rc) break;
        hipLaunchKernelGGL(fence_chain, dim3(1), wave, 0, s, static_cast<uint4 *>(words.p),
                           iterations, r);
        rc = launch_ok();
        break;
    }
    default:
        rc = SIFAR_EINVAL;
    }
    uint64_t h[R_WORDS] = {};
    if (!rc) rc = hip_ok(hipMemcpyAsync(h, r, sizeof(h), hipMemcpyDeviceToHost, s));
    if (!rc) rc = hip_ok(hipStreamSynchronize(s));
    if (rc) return rc;
    const bool pp = kind == SIFAR_FLOOR_PINGPONG_XCD || kind == SIFAR_FLOOR_PINGPONG_SAME_XCD;
    const bool ok = h[R_OK] == 1 && !(pp && h[R_SINK] != 0);
    info[0] = ok ? 1u : 0u;
    info[1] = static_cast<uint32_t>(h[R_XCC_A]);
    info[2] = static_cast<uint32_t>(h[R_XCC_B]);
    if (!ok) return SIFAR_EDEVICE;
    const double ticks = static_cast<double>(h[R_T1] - h[R_T0]);
    const double ops = pp ? 2.0 * iterations : static_cast<double>(iterations);
    *ns_per_op = ticks * 1e6 / static_cast<double>(khz) / ops;
    return SIFAR_OK;
}
