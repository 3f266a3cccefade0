// Host runtime behind the C ABI of include/sifar.h: configuration checks,
// library-owned device memory, host-side epoch accounting, eager launches and
// the captured decode-step graphs.
#include "sifar.h"

#include <hip/hip_runtime.h>

#include <map>
#include <new>

#include "sifar_kernels.h"

using namespace sifar;

struct sifar_ctx {
    sifar_config cfg{};
    int device = 0;
    int segs = 0;          // chunks per token
    int w_max = 0;         // max_tokens * segs
    int groups_per_token = 1;
    bool chain_grouping = false;  // persistent steps may use kChainGroupWaves-wave workgroups
    bool chain_prefetch = false;  // one-wave persistent steps' producers load sources ahead
    uint64_t slot_elems = 0;

    uint16_t *slots = nullptr;     // [N][2][slot_elems]
    uint32_t *stamps = nullptr;    // [2][w_max][N]
    uint32_t *consumed = nullptr;  // [2][w_max]
    uint32_t *produced = nullptr;  // [2][w_max]
    uint32_t *log = nullptr;       // [log_epochs][w_max]
    uint32_t *stamp_log = nullptr; // [log_epochs][w_max][2][N]
    uint16_t *stage = nullptr;     // [N][2][slot_elems]: late ranks' payload (deterministic injection)
    uint64_t *exch = nullptr;      // [kExchPlanes][max_tokens][exch_q]
    uint64_t *place = nullptr;     // [2][w_max] XCD tags of each chunk's consumer / producer
    int exch_q = 1;                // exchange words per token and parity
    DevState *state = nullptr;
    uint16_t *inject = nullptr;
    int32_t inject_entries = 0;
    bool slot_overrun = false;     // SIFAR_INJECT_SLOT_OVERRUN: no host dual-buffer limit

    uint32_t next_prod = 1, next_red = 1;
    int32_t prod_tokens[2] = {0, 0};
    uint32_t base_host = 0;        // epoch_base once all enqueued work has run
    bool poisoned = false;

    bool bound = false;
    sifar_step_buffers buf{};
    std::map<int32_t, hipGraphExec_t> graphs;
    hipStream_t capture = nullptr;
};

namespace {

constexpr int kVersion = 100;  // 0.1.0

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

template <typename T>
int dev_alloc(T **p, size_t count) {
    if (count == 0) count = 1;
    if (hipMalloc(reinterpret_cast<void **>(p), count * sizeof(T)) != hipSuccess) {
        *p = nullptr;
        return SIFAR_ENOMEM;
    }
    return SIFAR_OK;
}

int check_cfg(const sifar_config *c) {
    if (!c) return SIFAR_EINVAL;
    if (c->nranks < 1 || c->nranks > kMaxRanks) return SIFAR_EINVAL;
    if (c->hidden < 8 || c->hidden > 65536 || c->hidden % 8) return SIFAR_EINVAL;
    if (c->max_tokens < 1 || c->max_tokens > (1 << 20)) return SIFAR_EINVAL;
    if (c->reduces_per_step < 1 || c->reduces_per_step > (1 << 16)) return SIFAR_EINVAL;
    if (c->validate < SIFAR_VALIDATE_SPEC || c->validate > SIFAR_VALIDATE_NONE) return SIFAR_EINVAL;
    if (c->epilogue != 0 && c->epilogue != 1) return SIFAR_EINVAL;
    if (c->epilogue && !(c->rms_eps >= 0.0f)) return SIFAR_EINVAL;
    if (c->max_attempts < 1 || c->spin_limit < 1 || c->log_epochs < 1) return SIFAR_EINVAL;
    const int g = c->waves_per_group;
    if (g != 1 && g != 2 && g != 4 && g != 8 && g != 16) return SIFAR_EINVAL;
    if (c->fuse_peers != 0 && c->fuse_peers != 1) return SIFAR_EINVAL;
    if (c->persistent != 0 && c->persistent != 1) return SIFAR_EINVAL;
    if (c->buffers != 1 && c->buffers != 2) return SIFAR_EINVAL;
    // A persistent step reads slots its peers are writing at that moment. Only
    // ORDERED is sound there: without validation the reads race the writes,
    // and speculative loads issued with the stamp loads were measured to
    // return a rank's previous epoch while its stamp already read fresh (the
    // monotonicity the paper assumes, Sec. 8.1, does not hold across XCDs).
    if (c->persistent && c->validate != SIFAR_VALIDATE_ORDERED) return SIFAR_EINVAL;
    return SIFAR_OK;
}

void drop_graphs(sifar_t h) {
    for (auto &kv : h->graphs) (void)hipGraphExecDestroy(kv.second);
    h->graphs.clear();
}

Geometry geometry(const sifar_t h, int32_t tokens) {
    Geometry g{};
    g.nranks = h->cfg.nranks;
    g.tokens = tokens;
    g.hidden = h->cfg.hidden;
    g.segs = h->segs;
    g.w_max = h->w_max;
    g.slot_elems = h->slot_elems;
    return g;
}

int usable(const sifar_t h) {
    if (!h) return SIFAR_EINVAL;
    if (h->poisoned) return SIFAR_ESTATE;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return SIFAR_EHIP;
    if (dev != h->device) return SIFAR_EINVAL;
    return SIFAR_OK;
}

ProduceArgs produce_args(const sifar_t h, int32_t tokens, EpochRef ep, const uint16_t *src,
                         int64_t entry_stride, int64_t rank_stride, int32_t entries) {
    ProduceArgs a{};
    a.geo = geometry(h, tokens);
    a.ep = ep;
    a.slots = h->slots;
    a.stamps = h->stamps;
    a.consumed = h->consumed;
    a.produced = h->produced;
    a.src = src;
    a.entry_stride = entry_stride;
    a.rank_stride = rank_stride;
    a.entries = entries;
    a.entries_div = make_div(static_cast<uint32_t>(entries));
    a.inject = h->inject;
    a.inject_entries = h->inject_entries;
    a.inject_div = make_div(static_cast<uint32_t>(h->inject_entries > 0 ? h->inject_entries : 1));
    a.stage = h->inject ? h->stage : nullptr;
    a.err = h->state->err;
    return a;
}

ReduceArgs reduce_args(const sifar_t h, int32_t tokens, EpochRef ep) {
    ReduceArgs a{};
    a.geo = geometry(h, tokens);
    a.ep = ep;
    a.slots = h->slots;
    a.stamps = h->stamps;
    a.consumed = h->consumed;
    a.log = h->log;
    a.stamp_log = h->stamp_log;
    a.log_epochs = h->cfg.log_epochs;
    a.log_div = make_div(static_cast<uint32_t>(h->cfg.log_epochs));
    a.max_attempts = h->cfg.max_attempts;
    a.forced_retries = h->cfg.forced_retries;
    a.spin_limit = h->cfg.spin_limit;
    a.inject = h->inject;
    a.inject_entries = h->inject_entries;
    a.inject_div = make_div(static_cast<uint32_t>(h->inject_entries > 0 ? h->inject_entries : 1));
    a.stage = h->inject ? h->stage : nullptr;
    a.exch = h->exch;
    a.groups_per_token = h->groups_per_token;
    a.exch_parity_stride = h->cfg.max_tokens * h->exch_q;
    a.eps = h->cfg.rms_eps;
    a.err = h->state->err;
    return a;
}

int hip_status(hipError_t e) { return e == hipSuccess ? SIFAR_OK : SIFAR_EHIP; }

// Slot parity of epoch g is g & parity_mask: dual buffering, or one slot.
uint32_t parity_mask(const sifar_t h) { return h->cfg.buffers == 2 ? 1u : 0u; }

int launch_red(sifar_t h, const ReduceArgs &ra, const ProduceArgs *next, hipStream_t s) {
    return hip_status(launch_reduce(ra, next, h->cfg.validate, h->cfg.epilogue != 0,
                                    h->cfg.waves_per_group, s));
}

// Waves per workgroup of a persistent step. Grouping lets one publication
// (and, for a cross-XCD pair, one release fence) cover 4 chunks, and the
// epilogue's groups share one exchange word. Measured on MI355X (payload
// sweep shapes, us per all-reduce, one-wave vs grouped): plain steps at 1024
// chunks 2.88 vs 2.87 (N = 8) and 1.25 vs 1.59 (N = 4), at 2048 chunks
// 1.58 vs 1.85 (N = 2), 3.05 vs 2.95 (N = 4) and 8.2 vs 7.9 (N = 8), at
// 4096 chunks 3.41 vs 3.64 (N = 2), 7.53 vs 7.99 (N = 4) and 15.3 vs 16.4
// (N = 8); with the epilogue (MoE, 512 chunks) 3.06 vs 2.80. So plain steps
// run one wave per workgroup, epilogue steps group from 512 chunks.
int chain_waves(const sifar_ctx *h, int32_t tokens) {
    const int64_t chunks = static_cast<int64_t>(tokens) * h->segs;
    return h->cfg.epilogue && h->chain_grouping && h->segs % kChainGroupWaves == 0 &&
                   chunks >= 512
               ? kChainGroupWaves
               : 1;
}

// Arguments of the persistent step kernel for `tokens` tokens; returns the
// workgroup width (waves) it runs with.
int chain_args(const sifar_t h, int32_t tokens, ChainArgs *ca) {
    const int L = h->cfg.reduces_per_step;
    const EpochRef ep{&h->state->epoch_base, 0, 0};
    *ca = ChainArgs{};
    ca->p = produce_args(h, tokens, ep, static_cast<const uint16_t *>(h->buf.src_pool),
                         h->buf.pool_entry_stride, h->buf.pool_rank_stride, h->buf.pool_entries);
    ca->r = reduce_args(h, tokens, ep);
    // a persistent step's late ranks write their payload on time and delay
    // only their stamps (late_delay): nothing is staged
    ca->p.stage = nullptr;
    ca->r.stage = nullptr;
    if (h->cfg.epilogue) {
        ca->r.residual = static_cast<uint16_t *>(h->buf.residual);
        ca->r.weight = static_cast<const uint16_t *>(h->buf.weight);
        ca->r.y = static_cast<uint16_t *>(h->buf.y_ring);
    } else {
        ca->r.out = static_cast<uint16_t *>(h->buf.out_ring);
    }
    const int waves = chain_waves(h, tokens);
    ca->r.groups_per_token = h->segs / waves;  // the epilogue's exchange width
    ca->reduces = L;
    ca->ring_stride = static_cast<uint64_t>(h->cfg.max_tokens) * h->cfg.hidden;
    ca->late_delay = h->cfg.late_delay;
    ca->epoch_base = &h->state->epoch_base;
    ca->advance = static_cast<uint32_t>(L + (L & 1));
    ca->done = &h->state->chain_done;
    ca->place = h->place;
    ca->parity_mask = parity_mask(h);
    return waves;
}

// Graph of a per-epoch step (persistent steps are one direct launch).
int capture_step(sifar_t h, int32_t tokens, hipGraphExec_t *out) {
    const int L = h->cfg.reduces_per_step;
    const uint32_t advance = static_cast<uint32_t>(L + (L & 1));
    const uint64_t ring = static_cast<uint64_t>(h->cfg.max_tokens) * h->cfg.hidden;
    hipStream_t s = h->capture;
    if (hipStreamBeginCapture(s, hipStreamCaptureModeThreadLocal) != hipSuccess) return SIFAR_EHIP;
    int rc = SIFAR_OK;
    auto node_args = [&](int i, ProduceArgs *pa, ReduceArgs *ra) {
        const EpochRef ep{&h->state->epoch_base, static_cast<uint32_t>(i + 1),
                          static_cast<uint32_t>((i + 1) & 1) & parity_mask(h)};
        *pa = produce_args(h, tokens, ep, static_cast<const uint16_t *>(h->buf.src_pool),
                           h->buf.pool_entry_stride, h->buf.pool_rank_stride, h->buf.pool_entries);
        *ra = reduce_args(h, tokens, ep);
        if (h->cfg.epilogue) {
            ra->residual = static_cast<uint16_t *>(h->buf.residual);
            ra->weight = static_cast<const uint16_t *>(h->buf.weight);
            ra->y = static_cast<uint16_t *>(h->buf.y_ring) + i * ring;
        } else {
            ra->out = static_cast<uint16_t *>(h->buf.out_ring) + i * ring;
        }
    };
    ProduceArgs pa{}, pn{};
    ReduceArgs ra{}, rn{};
    if (h->cfg.fuse_peers && h->cfg.buffers == 2) {
        node_args(0, &pa, &ra);
        rc = hip_status(launch_produce(pa, h->cfg.waves_per_group, s));
        for (int i = 0; i < L && rc == SIFAR_OK; ++i) {
            node_args(i, &pa, &ra);
            if (i + 1 < L) {
                node_args(i + 1, &pn, &rn);
                rc = launch_red(h, ra, &pn, s);
            } else {
                rc = launch_red(h, ra, nullptr, s);
            }
        }
    } else {
        for (int i = 0; i < L && rc == SIFAR_OK; ++i) {
            node_args(i, &pa, &ra);
            rc = hip_status(launch_produce(pa, h->cfg.waves_per_group, s));
            if (rc == SIFAR_OK) rc = launch_red(h, ra, nullptr, s);
        }
    }
    if (rc == SIFAR_OK) rc = hip_status(launch_advance(&h->state->epoch_base, advance, s));
    hipGraph_t graph = nullptr;
    const hipError_t e = hipStreamEndCapture(s, &graph);
    if (rc == SIFAR_OK && e != hipSuccess) rc = SIFAR_EHIP;
    if (rc == SIFAR_OK && hipGraphInstantiate(out, graph, nullptr, nullptr, 0) != hipSuccess)
        rc = SIFAR_EHIP;
    if (graph) (void)hipGraphDestroy(graph);
    return rc;
}

}  // namespace

extern "C" {

void sifar_config_default(sifar_config *c) {
    if (!c) return;
    c->nranks = 8;
    c->hidden = 4096;
    c->max_tokens = 8;
    c->reduces_per_step = 64;
    c->validate = SIFAR_VALIDATE_SPEC;
    c->epilogue = 0;
    c->rms_eps = 1e-6f;
    c->max_attempts = 1u << 20;
    c->forced_retries = 0;
    c->spin_limit = 1u << 20;
    c->log_epochs = 64;
    c->waves_per_group = 1;
    c->fuse_peers = 1;
    c->persistent = 0;
    c->late_delay = 8;
    c->buffers = 2;
}

int sifar_version(void) { return kVersion; }

const char *sifar_strerror(int code) {
    switch (code) {
        case SIFAR_OK: return "ok";
        case SIFAR_EINVAL: return "invalid argument";
        case SIFAR_ENOMEM: return "out of memory";
        case SIFAR_EHIP: return "HIP runtime error";
        case SIFAR_ESTATE: return "call out of protocol order, or handle poisoned";
        case SIFAR_EDEVICE: return "device latched an error";
    }
    return "unknown error";
}

int sifar_init(const sifar_config *cfg, sifar_t *out) {
    if (!out) return SIFAR_EINVAL;
    *out = nullptr;
    int rc = check_cfg(cfg);
    if (rc) return rc;
    sifar_t h = new (std::nothrow) sifar_ctx;
    if (!h) return SIFAR_ENOMEM;
    h->cfg = *cfg;
    if (hipGetDevice(&h->device) != hipSuccess) {
        delete h;
        return SIFAR_EHIP;
    }
    const sifar_config &c = h->cfg;
    h->segs = (c.hidden + kChunk - 1) / kChunk;
    h->w_max = c.max_tokens * h->segs;
    // slots start on 256-byte boundaries
    h->slot_elems = ((static_cast<uint64_t>(c.max_tokens) * c.hidden + 127) / 128) * 128;
    if (c.epilogue) {
        const int G = c.waves_per_group;
        h->groups_per_token = (h->segs + G - 1) / G;
        if (h->groups_per_token > kLanes || (c.persistent && h->segs > kLanes)) {
            delete h;
            return SIFAR_EINVAL;  // the exchange polls one word per lane
        }
        if (h->groups_per_token > 1) {
            const int cap = max_active_groups(c.nranks, c.validate, true, G);
            if (cap <= 0 || static_cast<int64_t>(c.max_tokens) * h->groups_per_token > cap) {
                delete h;
                return SIFAR_EINVAL;  // a token's groups must be co-resident
            }
        }
    }
    h->exch_q = c.persistent && h->segs > h->groups_per_token ? h->segs : h->groups_per_token;
    if (c.persistent) {
        // every consumer and producer wave of a step is resident at once
        // with the epilogue the grid pads the tokens to a multiple of 8 (one
        // XCD per token)
        const int64_t tokens = c.epilogue ? 8 * ((static_cast<int64_t>(c.max_tokens) + 7) / 8)
                                          : c.max_tokens;
        const int64_t waves = 2 * tokens * h->segs;
        // the prefetching producer holds two epochs' sources: it needs more
        // registers, so it runs wherever the step still fits with them
        const int pcap = max_active_chain_groups(c.nranks, c.validate, c.epilogue != 0, 1, true);
        h->chain_prefetch = pcap > 0 && waves <= pcap;
        const int cap = h->chain_prefetch
                            ? pcap
                            : max_active_chain_groups(c.nranks, c.validate, c.epilogue != 0, 1, false);
        if (cap <= 0 || waves > cap) {
            delete h;
            return SIFAR_EINVAL;
        }
        const int gcap = c.epilogue ? max_active_chain_groups(c.nranks, c.validate, true,
                                                              kChainGroupWaves, false)
                                    : 0;
        h->chain_grouping = c.nranks * kChainGroupWaves <= kLanes && gcap > 0 &&
                            waves / kChainGroupWaves <= gcap;
    }
    rc = SIFAR_OK;
    if (!rc) rc = dev_alloc(&h->slots, static_cast<size_t>(c.nranks) * 2 * h->slot_elems);
    if (!rc) rc = dev_alloc(&h->stamps, static_cast<size_t>(2) * h->w_max * c.nranks);
    if (!rc) rc = dev_alloc(&h->consumed, static_cast<size_t>(2) * h->w_max);
    if (!rc) rc = dev_alloc(&h->produced, static_cast<size_t>(2) * h->w_max);
    if (!rc) rc = dev_alloc(&h->log, static_cast<size_t>(c.log_epochs) * h->w_max);
    if (!rc)
        rc = dev_alloc(&h->stamp_log,
                       static_cast<size_t>(c.log_epochs) * h->w_max * 2 * c.nranks);
    if (!rc) rc = dev_alloc(&h->exch, static_cast<size_t>(kExchPlanes) * c.max_tokens * h->exch_q);
    if (!rc) rc = dev_alloc(&h->place, static_cast<size_t>(2) * h->w_max);
    if (!rc) rc = dev_alloc(&h->state, 1);
    if (!rc && hipStreamCreateWithFlags(&h->capture, hipStreamNonBlocking) != hipSuccess)
        rc = SIFAR_EHIP;
    if (!rc) {
        hipStream_t s = h->capture;
        const uint64_t slot_words = static_cast<uint64_t>(c.nranks) * 2 * h->slot_elems / 2;
        hipError_t e = launch_fill_u32(reinterpret_cast<uint32_t *>(h->slots), 0, slot_words, s);
        if (e == hipSuccess)
            e = launch_fill_u32(h->stamps, 0, static_cast<uint64_t>(2) * h->w_max * c.nranks, s);
        if (e == hipSuccess) e = launch_fill_u32(h->consumed, 0, static_cast<uint64_t>(2) * h->w_max, s);
        if (e == hipSuccess) e = launch_fill_u32(h->produced, 0, static_cast<uint64_t>(2) * h->w_max, s);
        if (e == hipSuccess)
            e = launch_fill_u32(h->log, 0, static_cast<uint64_t>(c.log_epochs) * h->w_max, s);
        if (e == hipSuccess)
            e = launch_fill_u32(h->stamp_log, 0,
                                static_cast<uint64_t>(c.log_epochs) * h->w_max * 2 * c.nranks, s);
        if (e == hipSuccess)
            e = launch_fill_u32(reinterpret_cast<uint32_t *>(h->exch), 0,
                                static_cast<uint64_t>(kExchPlanes) * c.max_tokens * h->exch_q * 2,
                                s);
        if (e == hipSuccess)
            e = launch_fill_u32(reinterpret_cast<uint32_t *>(h->place), 0,
                                static_cast<uint64_t>(2) * h->w_max * 2, s);
        if (e == hipSuccess)
            e = launch_fill_u32(reinterpret_cast<uint32_t *>(h->state), 0,
                                sizeof(DevState) / sizeof(uint32_t), s);
        if (e == hipSuccess) e = hipStreamSynchronize(s);
        if (e != hipSuccess) rc = SIFAR_EHIP;
    }
    if (rc) {
        sifar_destroy(h);
        return rc;
    }
    *out = h;
    return SIFAR_OK;
}

void sifar_destroy(sifar_t h) {
    if (!h) return;
    (void)hipDeviceSynchronize();
    drop_graphs(h);
    if (h->capture) (void)hipStreamDestroy(h->capture);
    (void)hipFree(h->slots);
    (void)hipFree(h->stamps);
    (void)hipFree(h->consumed);
    (void)hipFree(h->produced);
    (void)hipFree(h->log);
    (void)hipFree(h->stamp_log);
    (void)hipFree(h->stage);
    (void)hipFree(h->exch);
    (void)hipFree(h->place);
    (void)hipFree(h->state);
    (void)hipFree(h->inject);
    delete h;
}

int sifar_produce(sifar_t h, const void *src, int64_t src_rank_stride, int32_t tokens,
                  void *stream) {
    int rc = usable(h);
    if (rc) return rc;
    if (!src || !aligned16(src) || tokens < 1 || tokens > h->cfg.max_tokens) return SIFAR_EINVAL;
    if (src_rank_stride % 8 || src_rank_stride < static_cast<int64_t>(tokens) * h->cfg.hidden)
        return SIFAR_EINVAL;
    // every slot holds an unreduced epoch (unless a test forces the overwrite)
    if (!h->slot_overrun && h->next_prod - h->next_red >= static_cast<uint32_t>(h->cfg.buffers))
        return SIFAR_ESTATE;
    const uint32_t g = h->next_prod;
    const EpochRef ep{&h->state->zero, g, g & parity_mask(h)};
    ProduceArgs pa = produce_args(h, tokens, ep, static_cast<const uint16_t *>(src), 0,
                                  src_rank_stride, 1);
    rc = hip_status(launch_produce(pa, h->cfg.waves_per_group, static_cast<hipStream_t>(stream)));
    if (rc) return rc;
    h->prod_tokens[g & 1u] = tokens;
    h->next_prod = g + 1;
    return SIFAR_OK;
}

static int reduce_common(sifar_t h, int32_t tokens, void *stream, uint16_t *out, uint16_t *residual,
                         const uint16_t *weight, uint16_t *y) {
    const uint32_t g = h->next_red;
    if (g >= h->next_prod) return SIFAR_ESTATE;  // nothing produced to reduce
    if (tokens != h->prod_tokens[g & 1u]) return SIFAR_EINVAL;
    const EpochRef ep{&h->state->zero, g, g & parity_mask(h)};
    ReduceArgs ra = reduce_args(h, tokens, ep);
    ra.out = out;
    ra.residual = residual;
    ra.weight = weight;
    ra.y = y;
    int rc = launch_red(h, ra, nullptr, static_cast<hipStream_t>(stream));
    if (rc) return rc;
    h->next_red = g + 1;
    return SIFAR_OK;
}

int sifar_reduce(sifar_t h, void *out, int32_t tokens, void *stream) {
    int rc = usable(h);
    if (rc) return rc;
    if (h->cfg.epilogue) return SIFAR_EINVAL;
    if (!out || !aligned16(out) || tokens < 1 || tokens > h->cfg.max_tokens) return SIFAR_EINVAL;
    return reduce_common(h, tokens, stream, static_cast<uint16_t *>(out), nullptr, nullptr, nullptr);
}

int sifar_reduce_rmsnorm(sifar_t h, void *residual, const void *weight, void *y, int32_t tokens,
                         void *stream) {
    int rc = usable(h);
    if (rc) return rc;
    if (!h->cfg.epilogue) return SIFAR_EINVAL;
    if (!residual || !weight || !y || !aligned16(residual) || !aligned16(weight) || !aligned16(y))
        return SIFAR_EINVAL;
    if (tokens < 1 || tokens > h->cfg.max_tokens) return SIFAR_EINVAL;
    return reduce_common(h, tokens, stream, nullptr, static_cast<uint16_t *>(residual),
                         static_cast<const uint16_t *>(weight), static_cast<uint16_t *>(y));
}

int sifar_bind_step(sifar_t h, const sifar_step_buffers *b) {
    int rc = usable(h);
    if (rc) return rc;
    if (!b || !b->src_pool || !aligned16(b->src_pool) || b->pool_entries < 1) return SIFAR_EINVAL;
    const int64_t row = static_cast<int64_t>(h->cfg.max_tokens) * h->cfg.hidden;
    if (b->pool_rank_stride % 8 || b->pool_entry_stride % 8) return SIFAR_EINVAL;
    if (b->pool_rank_stride < row) return SIFAR_EINVAL;
    if (b->pool_entries > 1 && b->pool_entry_stride < b->pool_rank_stride * h->cfg.nranks)
        return SIFAR_EINVAL;
    if (h->cfg.epilogue) {
        if (!b->residual || !b->weight || !b->y_ring || b->out_ring) return SIFAR_EINVAL;
        if (!aligned16(b->residual) || !aligned16(b->weight) || !aligned16(b->y_ring))
            return SIFAR_EINVAL;
    } else {
        if (!b->out_ring || !aligned16(b->out_ring) || b->residual || b->weight || b->y_ring)
            return SIFAR_EINVAL;
    }
    drop_graphs(h);
    h->buf = *b;
    h->bound = true;
    return SIFAR_OK;
}

int sifar_step(sifar_t h, int32_t tokens, void *stream) {
    int rc = usable(h);
    if (rc) return rc;
    if (!h->bound) return SIFAR_ESTATE;
    if (tokens < 1 || tokens > h->cfg.max_tokens) return SIFAR_EINVAL;
    if (h->next_prod != h->next_red) return SIFAR_ESTATE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int L = h->cfg.reduces_per_step;
    // Graph nodes take parity (i + 1) & 1 for epoch base + i + 1: base must be even.
    uint32_t base = h->next_red - 1;
    base += base & 1u;
    if (h->cfg.persistent) {
        // A persistent step is one kernel: launched directly, since replaying a
        // one-node graph measured ~5 us more per step on MI355X.
        if (base != h->base_host) {
            rc = hip_status(launch_set_base(&h->state->epoch_base, base, s));
            if (rc) return rc;
        }
        ChainArgs ca{};
        const int waves = chain_args(h, tokens, &ca);
        rc = hip_status(
            launch_chain(ca, h->cfg.validate, h->cfg.epilogue != 0, waves, h->chain_prefetch, s));
        if (rc) return rc;
        h->base_host = base + static_cast<uint32_t>(L + (L & 1));
        h->next_prod = h->next_red = base + static_cast<uint32_t>(L) + 1;
        const uint32_t last = h->next_red - 1;
        h->prod_tokens[last & 1u] = tokens;
        h->prod_tokens[(last + 1) & 1u] = tokens;
        return SIFAR_OK;
    }
    auto it = h->graphs.find(tokens);
    hipGraphExec_t exec = nullptr;
    if (it == h->graphs.end()) {
        rc = capture_step(h, tokens, &exec);
        if (rc) return rc;
        h->graphs[tokens] = exec;
    } else {
        exec = it->second;
    }
    if (base != h->base_host) {
        rc = hip_status(launch_set_base(&h->state->epoch_base, base, s));
        if (rc) return rc;
        h->base_host = base;
    }
    if (hipGraphLaunch(exec, s) != hipSuccess) return SIFAR_EHIP;
    h->base_host = base + static_cast<uint32_t>(L + (L & 1));
    h->next_prod = h->next_red = base + static_cast<uint32_t>(L) + 1;
    const uint32_t last = h->next_red - 1;
    h->prod_tokens[last & 1u] = tokens;
    h->prod_tokens[(last + 1) & 1u] = tokens;
    return SIFAR_OK;
}

int sifar_set_injection(sifar_t h, const uint16_t *table, int32_t entries, int32_t mode) {
    int rc = usable(h);
    if (rc) return rc;
    if (mode == SIFAR_INJECT_OFF) {
        if (hipDeviceSynchronize() != hipSuccess) return SIFAR_EHIP;
        (void)hipFree(h->inject);
        h->inject = nullptr;
        h->inject_entries = 0;
        h->slot_overrun = false;
        drop_graphs(h);
        return SIFAR_OK;
    }
    if (mode != SIFAR_INJECT_DETERMINISTIC && mode != SIFAR_INJECT_SLOT_OVERRUN) return SIFAR_EINVAL;
    if (h->cfg.validate == SIFAR_VALIDATE_NONE) return SIFAR_EINVAL;
    if (mode == SIFAR_INJECT_SLOT_OVERRUN) {
        h->slot_overrun = true;
        return SIFAR_OK;
    }
    if (!table || entries < 1) return SIFAR_EINVAL;
    if (hipDeviceSynchronize() != hipSuccess) return SIFAR_EHIP;
    // where late ranks' payloads wait until they catch up (per-epoch launches)
    if (!h->stage) {
        rc = dev_alloc(&h->stage, static_cast<size_t>(h->cfg.nranks) * 2 * h->slot_elems);
        if (rc) return rc;
    }
    uint16_t *d = nullptr;
    rc = dev_alloc(&d, static_cast<size_t>(entries));
    if (rc) return rc;
    if (hipMemcpy(d, table, sizeof(uint16_t) * entries, hipMemcpyHostToDevice) != hipSuccess) {
        (void)hipFree(d);
        return SIFAR_EHIP;
    }
    (void)hipFree(h->inject);
    h->inject = d;
    h->inject_entries = entries;
    drop_graphs(h);
    return SIFAR_OK;
}

int sifar_log_geometry(sifar_t h, int32_t *log_epochs, int32_t *chunks_per_token, int32_t *w_max) {
    if (!h) return SIFAR_EINVAL;
    if (log_epochs) *log_epochs = h->cfg.log_epochs;
    if (chunks_per_token) *chunks_per_token = h->segs;
    if (w_max) *w_max = h->w_max;
    return SIFAR_OK;
}

int sifar_read_log(sifar_t h, uint32_t *host_dst, size_t words) {
    if (!h || !host_dst) return SIFAR_EINVAL;
    if (words > static_cast<size_t>(h->cfg.log_epochs) * h->w_max) return SIFAR_EINVAL;
    if (hipDeviceSynchronize() != hipSuccess) return SIFAR_EHIP;
    if (hipMemcpy(host_dst, h->log, words * sizeof(uint32_t), hipMemcpyDeviceToHost) != hipSuccess)
        return SIFAR_EHIP;
    return SIFAR_OK;
}

int sifar_read_stamp_log(sifar_t h, uint32_t *host_dst, size_t words) {
    if (!h || !host_dst) return SIFAR_EINVAL;
    if (words > static_cast<size_t>(h->cfg.log_epochs) * h->w_max * 2 * h->cfg.nranks)
        return SIFAR_EINVAL;
    if (hipDeviceSynchronize() != hipSuccess) return SIFAR_EHIP;
    if (hipMemcpy(host_dst, h->stamp_log, words * sizeof(uint32_t), hipMemcpyDeviceToHost) !=
        hipSuccess)
        return SIFAR_EHIP;
    return SIFAR_OK;
}

int sifar_epochs(sifar_t h, uint32_t *next_produce, uint32_t *next_reduce) {
    if (!h) return SIFAR_EINVAL;
    if (next_produce) *next_produce = h->next_prod;
    if (next_reduce) *next_reduce = h->next_red;
    return SIFAR_OK;
}

int sifar_error_info(sifar_t h, uint32_t info[4]) {
    if (!h || !info) return SIFAR_EINVAL;
    if (hipDeviceSynchronize() != hipSuccess) return SIFAR_EHIP;
    if (hipMemcpy(info, h->state->err, 4 * sizeof(uint32_t), hipMemcpyDeviceToHost) != hipSuccess)
        return SIFAR_EHIP;
    return SIFAR_OK;
}

int sifar_status(sifar_t h) {
    if (!h) return SIFAR_EINVAL;
    uint32_t info[4] = {0, 0, 0, 0};
    const int rc = sifar_error_info(h, info);
    if (rc) return rc;
    if (info[0] != 0) {
        h->poisoned = true;
        return SIFAR_EDEVICE;
    }
    return h->poisoned ? SIFAR_ESTATE : SIFAR_OK;
}

}  // extern "C"
