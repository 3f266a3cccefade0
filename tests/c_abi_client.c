/*
 * A C11 client that drives libsifar through its C ABI alone: no Python and no
 * PyTorch, only the HIP runtime for device memory. tests/test_gpu_c_client.py
 * loads it as a shared library, calls sifar_c_client() with an argument vector
 * and checks what it writes against the oracle (built with -DSIFAR_CLIENT_MAIN
 * it is also a standalone program with the same arguments):
 *
 *   c_abi_client N T H L PERSISTENT in.bin out.bin
 *
 * in.bin holds E source entries of N x T x H bf16 bit patterns (rank-major).
 * The program reduces entry e as epoch e + 1 with eager sifar_produce /
 * sifar_reduce calls, then binds the E entries as a step's source pool and
 * runs one decode step of L all-reduces (PERSISTENT 1: one persistent launch,
 * ORDERED validation; 0: a captured per-epoch graph, SPEC validation), then
 * reduces every entry once more with sifar_allreduce_noalloc (no handle, no
 * allocation). out.bin receives the E eager outputs, the L step outputs and
 * the E allocation-free outputs, T x H each.
 * Returns 0 on success, 2 on a bad argument or file, 1 when a HIP or libsifar
 * call fails (after printing which).
 */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include "sifar.h"

/* Every failure jumps to `done`, which frees what was allocated. */
#define CHECK_HIP(call)                                                           \
    do {                                                                          \
        hipError_t e_ = (call);                                                   \
        if (e_ != hipSuccess) {                                                   \
            fprintf(stderr, "%s failed: %s\n", #call, hipGetErrorString(e_));     \
            goto done;                                                            \
        }                                                                         \
    } while (0)

#define CHECK_SIFAR(call)                                                         \
    do {                                                                          \
        int r_ = (call);                                                          \
        if (r_ != SIFAR_OK) {                                                     \
            fprintf(stderr, "%s failed: %d (%s)\n", #call, r_, sifar_strerror(r_)); \
            goto done;                                                            \
        }                                                                         \
    } while (0)

int sifar_c_client(int argc, char **argv) {
    if (argc != 8) {
        fprintf(stderr, "usage: %s N T H L PERSISTENT in.bin out.bin\n", argv[0]);
        return 2;
    }
    const int n = atoi(argv[1]), t = atoi(argv[2]), hd = atoi(argv[3]), l = atoi(argv[4]);
    const int persistent = atoi(argv[5]);
    if (n < 1 || t < 1 || hd < 8 || l < 1) return 2;
    const size_t row = (size_t)t * hd;    /* elements of one rank's partial */
    const size_t entry = (size_t)n * row; /* elements of one source entry */

    int status = 1;
    uint16_t *host_in = NULL, *host_out = NULL, *src = NULL, *out = NULL;
    sifar_t h = NULL;
    FILE *f = fopen(argv[6], "rb");
    if (!f) return 2;
    long bytes = -1;
    if (fseek(f, 0, SEEK_END) == 0) bytes = ftell(f);
    if (bytes <= 0 || (size_t)bytes % (entry * 2) != 0 || fseek(f, 0, SEEK_SET) != 0) {
        fclose(f);
        return 2;
    }
    const size_t e_count = (size_t)bytes / (entry * 2);
    const size_t outs = 2 * e_count + (size_t)l;
    host_in = malloc((size_t)bytes);
    host_out = malloc(outs * row * 2);
    const int read_ok = host_in && host_out && fread(host_in, 1, (size_t)bytes, f) == (size_t)bytes;
    fclose(f);
    if (!read_ok) {
        status = 2;
        goto done;
    }

    CHECK_HIP(hipMalloc((void **)&src, (size_t)bytes));
    CHECK_HIP(hipMalloc((void **)&out, outs * row * 2));
    CHECK_HIP(hipMemcpy(src, host_in, (size_t)bytes, hipMemcpyHostToDevice));

    sifar_config cfg;
    sifar_config_default(&cfg);
    cfg.nranks = n;
    cfg.hidden = hd;
    cfg.max_tokens = t;
    cfg.reduces_per_step = l;
    cfg.persistent = persistent;
    cfg.validate = persistent ? SIFAR_VALIDATE_ORDERED : SIFAR_VALIDATE_SPEC;
    CHECK_SIFAR(sifar_init(&cfg, &h));

    /* eager epochs 1..E, on the null stream */
    for (size_t e = 0; e < e_count; ++e) {
        CHECK_SIFAR(sifar_produce(h, src + e * entry, (int64_t)row, t, NULL));
        CHECK_SIFAR(sifar_reduce(h, out + e * row, t, NULL));
    }
    CHECK_SIFAR(sifar_status(h));

    /* one decode step over the same entries as its source pool */
    sifar_step_buffers b = {0};
    b.src_pool = src;
    b.pool_entries = (int32_t)e_count;
    b.pool_entry_stride = (int64_t)entry;
    b.pool_rank_stride = (int64_t)row;
    b.out_ring = out + e_count * row;
    CHECK_SIFAR(sifar_bind_step(h, &b));
    CHECK_SIFAR(sifar_step(h, t, NULL));
    CHECK_HIP(hipDeviceSynchronize());
    CHECK_SIFAR(sifar_status(h));
    CHECK_HIP(hipMemcpy(host_out, out, outs * row * 2, hipMemcpyDeviceToHost));
    uint32_t next_prod = 0, next_red = 0;
    CHECK_SIFAR(sifar_epochs(h, &next_prod, &next_red));

    /* the allocation-free entry point: every entry once more, queued back to
       back on the null stream, after the step's outputs were copied out */
    uint16_t *na = out + (e_count + (size_t)l) * row;
    for (size_t e = 0; e < e_count; ++e)
        CHECK_SIFAR(sifar_allreduce_noalloc(src + e * entry, (int64_t)row, n, t, hd, na + e * row,
                                            NULL));
    CHECK_HIP(hipDeviceSynchronize());
    CHECK_HIP(hipMemcpy(host_out + (e_count + (size_t)l) * row, na, e_count * row * 2,
                        hipMemcpyDeviceToHost));

    f = fopen(argv[7], "wb");
    if (!f) {
        status = 2;
        goto done;
    }
    const int write_ok = fwrite(host_out, 2, outs * row, f) == outs * row;
    if (fclose(f) != 0 || !write_ok) {
        status = 2;
        goto done;
    }
    printf("ok epochs %u\n", next_red);
    status = 0;
done:
    if (h) sifar_destroy(h);
    if (src) (void)hipFree(src);
    if (out) (void)hipFree(out);
    free(host_in);
    free(host_out);
    return status;
}

#ifdef SIFAR_CLIENT_MAIN
int main(int argc, char **argv) { return sifar_c_client(argc, argv); }
#endif
