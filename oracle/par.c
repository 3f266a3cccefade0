/*
 * par.c -- TEST INFRASTRUCTURE ONLY (see oracle/__init__.py): a host-thread
 * driver that runs the oracle's own oracle_reduce (ref.c) on contiguous
 * slices of one all-reduce's elements at once, for the benchmark's
 * multi-core CPU baseline. It adds no arithmetic: every output element is
 * computed by oracle_reduce exactly as in a single-threaded call (the sum of
 * one element never spans two slices), so the result is bit-identical.
 */
#include <pthread.h>
#include <stddef.h>
#include <stdint.h>

void oracle_reduce(const uint16_t *x, int nranks, size_t rank_stride, size_t count,
                   uint16_t *out);

struct slice {
    const uint16_t *x;
    int nranks;
    size_t rank_stride, begin, end;
    uint16_t *out;
};

static void *run_slice(void *arg)
{
    const struct slice *s = (const struct slice *)arg;
    oracle_reduce(s->x + s->begin, s->nranks, s->rank_stride, s->end - s->begin,
                  s->out + s->begin);
    return NULL;
}

/* Reduce `count` elements of x[nranks][rank_stride] into out[count] on
 * `threads` threads (1..256), each a contiguous slice. Returns the number of
 * threads used, or -1 when a thread could not be started (the caller's
 * output is then incomplete). */
int oracle_reduce_threads(const uint16_t *x, int nranks, size_t rank_stride, size_t count,
                          uint16_t *out, int threads)
{
    enum { kMax = 256 };
    if (threads < 1) threads = 1;
    if (threads > kMax) threads = kMax;
    if ((size_t)threads > count) threads = count > 0 ? (int)count : 1;
    struct slice sl[kMax];
    pthread_t tid[kMax];
    int started = 0, ok = 1;
    for (int t = 0; t < threads; ++t) {
        sl[t].x = x;
        sl[t].nranks = nranks;
        sl[t].rank_stride = rank_stride;
        sl[t].begin = count * (size_t)t / (size_t)threads;
        sl[t].end = count * (size_t)(t + 1) / (size_t)threads;
        sl[t].out = out;
    }
    for (int t = 1; t < threads; ++t) {
        if (pthread_create(&tid[t], NULL, run_slice, &sl[t]) != 0) {
            ok = 0;
            break;
        }
        started = t;
    }
    run_slice(&sl[0]);
    for (int t = 1; t <= started; ++t) pthread_join(tid[t], NULL);
    return ok ? threads : -1;
}
