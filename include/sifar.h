/*
 * sifar.h -- C ABI of libsifar, a single-GPU (MI355X, gfx950) implementation of
 * the data path of SiFAR, the synchronization-free one-shot all-reduce
 * ("SiFAR: Synchronization-Free All-Reduce for Low-Latency LLM Inference").
 *
 * What one all-reduce computes (Sec. 3.1 "Oneshot", and the pull-and-reduce
 * listing of Sec. 4.2): every rank's partial hidden state is pulled and added,
 * peer after peer in ascending rank order. Here payloads are bf16, the sum is
 * accumulated in fp32 (IEEE adds, round to nearest even, subnormals kept) and
 * rounded once to bf16, round to nearest even.
 *
 * How it is synchronised:
 *  - No bottom barrier (Sec. 3.3, 4.1 "Dual Buffering Design"): every rank
 *    owns two payload slots and two flag ("stamp") slots and alternates
 *    between them; epoch g uses parity g & 1, so a slot is rewritten only after
 *    the reduction two epochs back, which stream order has completed.
 *  - No top barrier (Sec. 3.5, 4.1 "Speculative Reduction Design", 4.2
 *    "Speculative Reduction"): the reduction loads the payload without
 *    waiting, validates each rank's stamp against the epoch afterwards, and
 *    re-runs on a stale stamp. The flag of epoch g is g itself (the paper's
 *    flag grows by one per all-reduce; Sec. 4.2 "Verification Logic
 *    Correctness"). The paper compares the SUM of the flags with N * flag;
 *    this library compares each rank's stamp with g (equivalent under dual
 *    buffering, and it names the stale ranks).
 *
 * The N ranks are emulated on one GPU: each rank's slots are HBM buffers, and
 * a producer kernel plays the peers, copying each rank's partial into its slot
 * and then storing its stamp after it. One process, one GPU; nothing crosses a
 * device boundary.
 *
 * Conventions
 *  - Every function returns int: SIFAR_OK (0) or a negative SIFAR_E* code.
 *    Nothing aborts, throws or prints.
 *  - Device pointers are HIP device addresses on the handle's device, 16-byte
 *    aligned. bf16 values are passed as raw 16-bit patterns. Host pointers are
 *    ordinary host memory.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *    Enqueueing calls are asynchronous and stream-ordered; only sifar_status()
 *    and sifar_read_log() synchronise.
 *  - The library owns the slots, stamps, counters, decision log, injection
 *    table, error word and captured graphs. The caller owns every buffer it
 *    passes in and must keep it alive until the enqueued work has finished.
 *  - One host thread per handle. Calls on one handle must use one stream, or
 *    streams the caller orders.
 *  - A device-detected error (retry budget exhausted, slot rewritten before
 *    it was consumed, epilogue exchange timed out) is latched in device memory
 *    and reported by the next sifar_status() as SIFAR_EDEVICE; the handle then
 *    refuses further work (SIFAR_ESTATE) until destroyed.
 */
#ifndef SIFAR_H
#define SIFAR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct sifar_ctx *sifar_t;

/* ---- return codes --------------------------------------------------------- */
#define SIFAR_OK 0
#define SIFAR_EINVAL (-1)  /* bad argument; nothing was enqueued */
#define SIFAR_ENOMEM (-2)  /* device or host allocation failed */
#define SIFAR_EHIP (-3)    /* a HIP runtime call failed */
#define SIFAR_ESTATE (-4)  /* call out of protocol order, or handle poisoned */
#define SIFAR_EDEVICE (-5) /* the device latched an error (see sifar_error_info) */

/* device error kinds (sifar_error_info, info[0]) */
#define SIFAR_DEV_RETRY_BUDGET 1 /* a chunk exhausted max_attempts: its stamps never became fresh */
#define SIFAR_DEV_WAW 2          /* producer found a slot whose previous epoch was not consumed */
#define SIFAR_DEV_EXCHANGE 3     /* epilogue: a token's segments did not all arrive within spin_limit */

/* ---- validation modes ------------------------------------------------------
 * SPEC     the paper's speculative reduction (Sec. 3.5, 4.2): payload and
 *          stamps are loaded together, validation follows, a stale stamp
 *          re-runs both. Correct when a rank whose stamp is fresh at
 *          validation also had its payload in place when it was loaded -- the
 *          monotonicity assumption of Sec. 8.1. It holds for the per-epoch
 *          launches (eager calls, step graphs with persistent = 0): every
 *          epoch's payload was written by an earlier launch. It does not hold
 *          for a producer that is writing at that moment: measured on MI355X
 *          with producer and consumer on different XCDs, ~2 % of persistent
 *          all-reduces accepted a rank's previous epoch under a fresh stamp
 *          (sifar_litmus measures the same per handoff). So persistent steps
 *          refuse SPEC (SIFAR_EINVAL).
 * ORDERED  stamps are read first and the payload is loaded only once all
 *          are fresh: a top barrier by flag polling (the "oneshot + dual
 *          buffering" configuration of Sec. 3.4). Correct without any
 *          monotonicity assumption; the only mode of persistent steps.
 * NONE     no stamps are read: the idealised "no barrier" configuration of
 *          Sec. 6.3. Only correct when stream order alone guarantees the data,
 *          so not allowed with persistent steps. */
#define SIFAR_VALIDATE_SPEC 0
#define SIFAR_VALIDATE_ORDERED 1
#define SIFAR_VALIDATE_NONE 2

/* ---- stale-stamp injection ---------------------------------------------------
 * DETERMINISTIC: for epoch g, table entry (g - 1) % entries holds two rank masks:
 *   bits 0-7  late ranks. Per-epoch launches: the producer writes their
 *             payload into a library-owned stage, not their slot (which keeps
 *             the rank's previous epoch), and writes no stamp; right after the
 *             reduction's first failed validation of each chunk the rank
 *             "catches up": its payload moves into the slot and, after a
 *             release, its stamp is written, so the retry must reload the
 *             payload. Persistent steps: the payload is written on time and
 *             the stamp lands late_delay sleeps later.
 *   bits 8-15 withheld ranks: the stamp is never written; the chunk exhausts
 *             max_attempts and SIFAR_DEV_RETRY_BUDGET is latched.
 * The resulting per-chunk decisions are exactly predictable (see the log). */
#define SIFAR_INJECT_OFF 0
#define SIFAR_INJECT_DETERMINISTIC 1
/* SLOT_OVERRUN: the host stops refusing a sifar_produce that would rewrite a
 * slot whose epoch has not been reduced yet (the dual-buffer limit, Sec. 4.1),
 * so a test can force the write-after-write hazard that dual buffering
 * removes. The producer kernel's own check must then latch SIFAR_DEV_WAW, and
 * the overwritten epoch's reduction sees fresh stamps of another epoch, so it
 * exhausts max_attempts. `table` and `entries` are ignored; an installed
 * DETERMINISTIC table stays installed. Eager calls only (a step needs every
 * produced epoch reduced first). SIFAR_INJECT_OFF ends it. */
#define SIFAR_INJECT_SLOT_OVERRUN 2

/* ---- configuration ---------------------------------------------------------- */
typedef struct {
    int32_t nranks;           /* N: emulated tensor-parallel ranks, 1..8 */
    int32_t hidden;           /* H: elements per token, multiple of 8, 8..65536 */
    int32_t max_tokens;       /* T_max: largest batch (tokens per all-reduce), >= 1 */
    int32_t reduces_per_step; /* L: all-reduces in one decode step (2 per layer, Sec. 2.4), >= 1 */
    int32_t validate;         /* SIFAR_VALIDATE_* */
    int32_t epilogue;         /* 0: plain all-reduce; 1: fused residual-add + RMSNorm */
    float rms_eps;            /* RMSNorm epsilon (epilogue only) */
    uint32_t max_attempts;    /* retry budget per chunk (Sec. 4.2's loop is unbounded), >= 1 */
    uint32_t forced_retries;  /* treat the first k validations as failed (Sec. 6.3 forced-retry measurement) */
    uint32_t spin_limit;      /* bound on the epilogue's cross-segment wait, in polls, >= 1 */
    int32_t log_epochs;       /* decision-log ring length, in epochs, >= 1 */
    int32_t waves_per_group;  /* waves (64 lanes) per workgroup: 1, 2, 4, 8 or 16 */
    int32_t fuse_peers;       /* step graphs: 1 = the launch reducing epoch g also writes the
                                 peers' epoch g + 1 (other parity); 0 = separate producer and
                                 reduction launches */
    int32_t persistent;       /* step graphs: 1 = one persistent launch runs the whole step, its
                                 consumer waves and the emulated peers' waves synchronising
                                 through stamps in flight (a megakernel-style chain, Sec. 5);
                                 needs validate = ORDERED and 2 x max_tokens x
                                 ceil(hidden / 512) co-resident waves */
    uint32_t late_delay;      /* persistent steps with injection: a late rank's stamp lands
                                 this many ~0.2 us sleeps after its payload */
    int32_t buffers;          /* 2: dual buffering (Sec. 3.3; no bottom barrier). 1: one slot per
                                 rank, rewritten only after the previous all-reduce has finished
                                 reading it -- the bottom barrier of Sec. 3.1, for the ablation
                                 (no fused peers; the producer may not run ahead) */
} sifar_config;

/* Fills cfg with: N=8, H=4096, T_max=8, L=64, SPEC, no epilogue, eps=1e-6,
 * max_attempts=1<<20, forced_retries=0, spin_limit=1<<20, log_epochs=64,
 * waves_per_group=1, fuse_peers=1, persistent=0, late_delay=8, buffers=2. Never
 * fails. */
void sifar_config_default(sifar_config *cfg);

/* Library version: major * 10000 + minor * 100 + patch. */
int sifar_version(void);

/* Create a handle on the current HIP device. Validates cfg (SIFAR_EINVAL),
 * allocates the library-owned device state and zeroes it (all stamps 0 =
 * stale for every epoch g >= 1). *out receives the handle on success, NULL on
 * failure. */
int sifar_init(const sifar_config *cfg, sifar_t *out);

/* Release everything the handle owns (synchronises the device first). NULL is a
 * no-op. */
void sifar_destroy(sifar_t h);

/* ---- eager calls: one epoch at a time ---------------------------------------
 * Epochs are numbered from 1. The producer may run at most one epoch ahead of
 * the reduction: that is all two slots allow (Sec. 3.3); a third produce
 * before a reduce returns SIFAR_ESTATE (with buffers = 1, a second one). */

/* The emulated peers write epoch g = next produced epoch. Rank r's partial is
 * read from src + r * src_rank_stride (elements), laid out [tokens][hidden]
 * bf16, and copied into rank r's slot of parity g & 1; then rank r's stamps of
 * every chunk are set to g, ordered after the payload within the producing
 * wave and published device-wide by the end of the launch (Sec. 4.1: a rank
 * raises its flag only once its partial is in the payload buffer), except for
 * ranks the injection table marks late or withheld.
 * 1 <= tokens <= max_tokens; src_rank_stride >= tokens * hidden, multiple of 8. */
int sifar_produce(sifar_t h, const void *src, int64_t src_rank_stride, int32_t tokens,
                  void *stream);

/* Reduce the oldest produced, unreduced epoch into out[tokens][hidden] bf16.
 * tokens must equal the producer's. Requires epilogue == 0. */
int sifar_reduce(sifar_t h, void *out, int32_t tokens, void *stream);

/* Reduce the oldest produced epoch and apply the fused epilogue. With a the
 * all-reduce result rounded to bf16 (not stored):
 *   residual[t][h] <- bf16( a + residual )                   (in place)
 *   y[t][h]         = bf16( residual * w[h] / sqrt(mean_h(residual^2) + eps) )
 * The paper does not describe this epilogue; it is the operation that follows
 * each all-reduce of a pre-norm transformer layer. residual: [tokens][hidden],
 * weight: [hidden], y: [tokens][hidden], all bf16. Requires epilogue == 1. */
int sifar_reduce_rmsnorm(sifar_t h, void *residual, const void *weight, void *y,
                         int32_t tokens, void *stream);

/* ---- decode step: L chained all-reduces in one captured HIP graph -----------
 * Binds the caller-owned buffers a step graph uses (Sec. 6.1 times
 * all-reduces back to back inside the forward pass; Sec. 3.5: a CUDA graph
 * or megakernel keeps the GPUs in lockstep). Rebinding drops captured graphs.
 *   src_pool      [pool_entries][N][...] bf16: epoch g's partials are entry
 *                 (g - 1) % pool_entries; rank r at offset r * pool_rank_stride,
 *                 [tokens][hidden] inside; entries pool_entry_stride apart.
 *   out_ring      plain: [L][max_tokens][hidden]; node i writes out_ring[i]
 *   residual,
 *   weight, y_ring  epilogue: residual [max_tokens][hidden] (updated in place,
 *                 chained across the L reduces), weight [hidden], y_ring
 *                 [L][max_tokens][hidden]; node i writes y_ring[i].
 * Unused pointers must be NULL. Strides are in elements, multiples of 8. */
typedef struct {
    const void *src_pool;
    int32_t pool_entries;
    int64_t pool_entry_stride;
    int64_t pool_rank_stride;
    void *out_ring;
    void *residual;
    const void *weight;
    void *y_ring;
} sifar_step_buffers;

int sifar_bind_step(sifar_t h, const sifar_step_buffers *b);

/* Enqueue one decode step for `tokens` tokens: L all-reduces plus one
 * epoch-counter advance. Per-epoch steps are one hipGraphLaunch: with
 * fuse_peers the graph is produce(g1), then L-1 launches that each reduce g_i
 * while writing g_(i+1), then reduce(g_L): L + 1 kernel nodes; without it,
 * L x (produce, reduce). A persistent step is one kernel launch for the whole
 * step (a one-node graph replay measured slower). In a persistent step the
 * peers run concurrently with the reduction, so a reduction often reaches an
 * epoch before its stamps (the decision log records the polls: attempts and
 * the stale ranks of the first and last poll), and injected late stamps land
 * after late_delay instead of after the first failed validation.
 * A per-epoch step's graph for a token count is captured on first use (on a
 * library-owned stream) and replayed afterwards; epochs and parities come
 * from a device-resident counter, so neither a replay nor a persistent
 * launch needs per-all-reduce host work. Requires no produced-but-unreduced
 * epoch (SIFAR_ESTATE).
 * A persistent step needs all its waves resident at once (checked at init
 * against an otherwise idle GPU); persistent steps of several handles that run
 * concurrently on different streams may not fit together, and then end with a
 * latched SIFAR_EDEVICE (every wait is bounded) instead of completing. Once one
 * wave of a persistent step has latched an error, the others end within
 * microseconds: a wait that has lasted 64 polls also reads the error word. */
int sifar_step(sifar_t h, int32_t tokens, void *stream);

/* ---- injection, logs, state --------------------------------------------------- */

/* Install (copies) a host table of `entries` uint16 words (late | withheld << 8)
 * for `mode` DETERMINISTIC, or switch on SLOT_OVERRUN; SIFAR_INJECT_OFF clears
 * both. Rank bits >= N are ignored. Drops captured graphs. Not allowed with
 * SIFAR_VALIDATE_NONE. */
int sifar_set_injection(sifar_t h, const uint16_t *table, int32_t entries, int32_t mode);

/* Decision log geometry: the log is a ring of log_epochs rows of w_max words;
 * epoch g, chunk c -> word ((g - 1) % log_epochs) * w_max + c. A chunk is the
 * 512 elements [t][s*512, s*512+512) of token t (the last of a row may be
 * shorter); c = t * chunks_per_token + s. */
int sifar_log_geometry(sifar_t h, int32_t *log_epochs, int32_t *chunks_per_token,
                       int32_t *w_max);

/* Copy the decision log to host memory (synchronises the device). Each word:
 * bits 0-15 attempts (saturating), 16-23 stale-rank mask of the first
 * validation, 24-31 stale-rank mask of the last one. An attempt is one
 * validation: in per-epoch launches a load of stamps and payload, in a
 * persistent step one poll of the stamps. `words` must be at most
 * log_epochs * w_max. */
int sifar_read_log(sifar_t h, uint32_t *host_dst, size_t words);

/* Copy the raw-stamp log to host memory (synchronises the device). Beside
 * each decision word the library keeps the N stamps the chunk's first and
 * last validation saw, so that every logged stale-rank mask can be
 * recomputed from them (Sec. 4.2: validation compares each rank's flag with
 * the epoch; Sec. 6.3 measures the mis-speculation rate). Same ring as the
 * decision log: epoch g, chunk c, validation v (0 first, 1 last), rank r ->
 * word (((g - 1) % log_epochs) * w_max + c) * 2N + v * N + r. In NONE mode no
 * stamp is read and the words are 0. `words` must be at most
 * log_epochs * w_max * 2N. */
int sifar_read_stamp_log(sifar_t h, uint32_t *host_dst, size_t words);

/* Next epoch to produce and next epoch to reduce (host-side accounting). */
int sifar_epochs(sifar_t h, uint32_t *next_produce, uint32_t *next_reduce);

/* Synchronise the device and check the device error word: SIFAR_OK, or
 * SIFAR_EDEVICE (and the handle is poisoned). */
int sifar_status(sifar_t h);

/* After SIFAR_EDEVICE: info[0] kind (SIFAR_DEV_*), info[1] epoch, info[2]
 * chunk, info[3] attempts. Synchronises. */
int sifar_error_info(sifar_t h, uint32_t info[4]);

/* Static string for a return code. */
const char *sifar_strerror(int code);

/* ---- Latency floors --------------------------------------------------------
 * The yardsticks a small all-reduce is read against (the paper times its
 * all-reduces back to back inside one persistent kernel to leave launch
 * overhead out, Sec. 6.1; on one GPU the launch gap and the cost of one
 * coherent memory round trip are what a small all-reduce is made of).
 * Needs no handle. Each kind measures `iterations` operations and writes the
 * mean nanoseconds per operation to *ns_per_op:
 *
 *  GRAPH_NODE        a captured hipGraph of `iterations` empty one-wave
 *                    kernels, replayed; ns per node (iterations <= 4096)
 *  EAGER_LAUNCH      `iterations` eager launches of the same kernel; ns each
 *                    (iterations <= 4096)
 *  ATOMIC            dependent agent-scope fetch-and-add on one word
 *  ACQUIRE_LOAD      dependent agent-scope acquire loads of one word (a load
 *                    plus the L2 invalidate that acquire implies)
 *  COHERENT_LOAD     dependent agent-scope relaxed loads of one word
 *  WARM_LOAD         dependent loads walking a 1 MiB ring that one pass has
 *                    just read, a new 128-byte line each hop (more than the
 *                    CU's L1 holds, far less than the XCD's L2)
 *  COLD_LOAD         dependent loads over a 1 GiB ring, each in a new line
 *                    and a new 4 MiB region, after the ring was pushed out of
 *                    L2 and the Infinity Cache (misses every cache and the
 *                    translation caches; iterations <= 65536)
 *  RELEASE_FENCE     a 16-byte store followed by an agent-scope release fence
 *  PINGPONG_XCD      one-way release -> acquire handoff between two waves on
 *                    different XCDs (iterations round trips, <= 65536)
 *  PINGPONG_SAME_XCD the same between two waves on one XCD
 *
 * info[0] is 1 when the probe completed, info[1] and info[2] the XCD (XCC_ID)
 * the probe's first and second wave ran on (0 for host-timed kinds).
 * Synchronises `stream`; allocates and frees its own device memory (1.5 GiB
 * for COLD_LOAD). Returns SIFAR_EINVAL for an unknown kind, a null pointer or
 * iterations out of range, SIFAR_ENOMEM, SIFAR_EHIP, or SIFAR_EDEVICE when a
 * handoff's bounded wait gave up (the partner wave never answered). */
enum {
    SIFAR_FLOOR_GRAPH_NODE = 0,
    SIFAR_FLOOR_EAGER_LAUNCH = 1,
    SIFAR_FLOOR_ATOMIC = 2,
    SIFAR_FLOOR_ACQUIRE_LOAD = 3,
    SIFAR_FLOOR_COHERENT_LOAD = 4,
    SIFAR_FLOOR_WARM_LOAD = 5,
    SIFAR_FLOOR_COLD_LOAD = 6,
    SIFAR_FLOOR_RELEASE_FENCE = 7,
    SIFAR_FLOOR_PINGPONG_XCD = 8,
    SIFAR_FLOOR_PINGPONG_SAME_XCD = 9
};
int sifar_floor(int32_t kind, int32_t iterations, void *stream, double *ns_per_op,
                uint32_t info[4]);

/* ---- Handoff litmus --------------------------------------------------------
 * Checks the memory-model assumption the validation rests on (Sec. 4.2: a
 * fresh stamp must imply fresh payload; Sec. 8.1 argues it for read-first
 * loads) on this GPU. `pairs` producer/consumer wave pairs (a multiple of 8,
 * 8..512) each pass one dual-buffered slot of 8 ranks x 64 lanes x 16 bytes
 * through `trials` epochs (1..2^20), with the persistent step's primitives and
 * slot discipline; the consumer compares every word it accepted with the epoch
 * it validated.
 *
 *  protocol  SIFAR_LITMUS_ORDERED: stamps first, then (from another XCD) an
 *            acquire, then the payload -- the persistent step's reader;
 *            SIFAR_LITMUS_READ_FIRST: payload and stamps loaded together and
 *            accepted when every stamp is fresh -- the paper's speculative
 *            reader (a stale stamp leads to an acquire and a reload of both);
 *            SIFAR_LITMUS_ORDERED_PREFETCH: the ORDERED reader against a
 *            producer that publishes as the persistent step's prefetching
 *            producer does: buffer stores of the slot, buffer loads of the
 *            next epoch's sources, a wait until only those loads are
 *            outstanding (on one XCD; a release fence across XCDs), then the
 *            flags. The other two protocols' producer stores the slot and
 *            waits for everything it has outstanding.
 *  placement SIFAR_LITMUS_CROSS_XCD: producer and consumer on different XCDs;
 *            SIFAR_LITMUS_SAME_XCD: on one XCD (workgroups are dealt to the 8
 *            XCDs round robin; the waves read where they actually ran)
 *
 * On return *result holds the trials completed, the trials whose accepted
 * payload held a word of another epoch (violations), how many of those were
 * in the first two epochs (where the stale words are the slot's initial
 * zeros rather than a rewritten epoch's), the bounded waits that
 * gave up, how many pairs landed as asked, the consumers' mean nanoseconds per
 * trial, and for the first violation {epoch, word found, word expected,
 * (producer XCD << 8) | consumer XCD}. Synchronises `stream`; allocates and
 * frees its own device memory (24 KiB per pair plus control words). Returns
 * SIFAR_EINVAL for a bad argument, SIFAR_ENOMEM, SIFAR_EHIP, or SIFAR_EDEVICE
 * when a wait gave up (the result is still filled in). Violations are data,
 * not an error. */
#define SIFAR_LITMUS_ORDERED 0
#define SIFAR_LITMUS_READ_FIRST 1
#define SIFAR_LITMUS_ORDERED_PREFETCH 2
#define SIFAR_LITMUS_CROSS_XCD 0
#define SIFAR_LITMUS_SAME_XCD 1
typedef struct {
    uint64_t trials;
    uint64_t violations;
    uint64_t violations_first_epochs;
    uint64_t timeouts;
    uint32_t pairs_placed;
    uint32_t pairs;
    double ns_per_trial;
    uint32_t first_bad[4];
} sifar_litmus_result;
int sifar_litmus(int32_t protocol, int32_t placement, int32_t pairs, int32_t trials,
                 void *stream, sifar_litmus_result *result);

/* ---- Allocation-free all-reduce ---------------------------------------------
 * For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc. One
 * all-reduce of `tokens` x `hidden` bf16 over `nranks` emulated ranks, the work
 * of sifar_produce followed by sifar_reduce on a SIFAR_VALIDATE_SPEC handle,
 * without a handle: the emulated peers copy rank r's partial
 * (src + r * src_rank_stride elements, laid out [tokens][hidden]) into a slot
 * and stamp it with the call's epoch, then the speculative reduction
 * validates the stamps and writes the fixed-order fp32 sum, rounded to bf16,
 * to out[tokens][hidden]. Two kernel launches on `stream`; nothing is
 * allocated or freed (no hipMalloc, hipFree or other allocating call), and
 * nothing synchronises.
 *
 * Scratch: the library's state for this call (slots, stamps, consumed and
 * produced words, decision log, epoch and error words) lives in one static
 * device array of SIFAR_NOALLOC_SCRATCH_BYTES per GPU, held from the first
 * call on that GPU until the process ends. Every call on a GPU shares that
 * GPU's array and leaves its contents behind; epochs grow from call to call
 * (host-side count per device), so a stamp of an earlier call is always
 * stale. Calls that overlap on one GPU (other streams, other host threads
 * without ordering) race on the array and may return wrong sums; calls
 * ordered on one stream never do, and then the producer's launch completes
 * before the reduction's, so no validation fails and no device error arises.
 *
 * Limits: 1 <= nranks <= 8; hidden a multiple of 8 in 8..65536;
 * 1 <= tokens <= SIFAR_NOALLOC_MAX_TOKENS; tokens * hidden <=
 * SIFAR_NOALLOC_MAX_ELEMS (512 KiB of bf16 per rank: 64 tokens x 4096);
 * src_rank_stride >= tokens * hidden and a multiple of 8; src and out 16-byte
 * aligned device pointers on the current device. Anything else returns
 * SIFAR_EINVAL before any work is enqueued; SIFAR_EHIP if a launch or the
 * symbol lookup fails. */
#define SIFAR_NOALLOC_MAX_TOKENS 64
#define SIFAR_NOALLOC_MAX_ELEMS 262144
#define SIFAR_NOALLOC_SCRATCH_BYTES 8437248 /* 8 MiB of slots + 47.5 KiB of words */
int sifar_allreduce_noalloc(const void *src, int64_t src_rank_stride, int32_t nranks,
                            int32_t tokens, int32_t hidden, void *out, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* SIFAR_H */
