/*
 * A C consumer of the GoCkpt C ABI: no Python, no torch, only the HIP runtime
 * API for device memory and streams.  Reads seeded inputs from a file, runs
 * one K-step save window (Sec. 4.2.1), drains, restores on the host (Sec.
 * 4.3.1) and writes the restored checkpoint and the device state back out for
 * the test to compare with the CPU oracle.
 *
 *   window_c <in.bin> <out.bin>
 *   in.bin:  int64 n, int64 K, int64 bounds[K+1], float p0[n],
 *            uint16 grads[K][n] (bf16 bits)
 *   out.bin: float p[n], m[n], v[n] (restored), uint16 w[n] (restored),
 *            float p_dev[n] (device master after step K), int64 t
 */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "gockpt.h"

#define CHECK_HIP(x)                                                              \
    do {                                                                          \
        hipError_t e_ = (x);                                                      \
        if (e_ != hipSuccess) {                                                   \
            fprintf(stderr, "%s:%d %s: %s\n", __FILE__, __LINE__, #x, hipGetErrorString(e_)); \
            return 2;                                                             \
        }                                                                         \
    } while (0)

#define CHECK_G(ctx, x)                                                           \
    do {                                                                          \
        int rc_ = (x);                                                            \
        if (rc_ < 0) {                                                            \
            fprintf(stderr, "%s:%d %s -> %d: %s\n", __FILE__, __LINE__, #x, rc_, gockpt_last_error(ctx)); \
            return 3;                                                             \
        }                                                                         \
    } while (0)

static int read_all(FILE* f, void* p, size_t bytes) { return fread(p, 1, bytes, f) == bytes ? 0 : -1; }

int main(int argc, char** argv) {
    if (argc != 3) {
        fprintf(stderr, "usage: %s in.bin out.bin\n", argv[0]);
        return 1;
    }
    FILE* f = fopen(argv[1], "rb");
    if (!f) return 1;
    int64_t n = 0, K = 0;
    if (read_all(f, &n, 8) || read_all(f, &K, 8) || n <= 0 || K < 1 || K > GOCKPT_MAX_K) return 1;
    int64_t* bounds = malloc((size_t)(K + 1) * 8);
    float* p0 = malloc((size_t)n * 4);
    uint16_t* grads = malloc((size_t)(K * n) * 2);
    if (!bounds || !p0 || !grads) return 1;
    if (read_all(f, bounds, (size_t)(K + 1) * 8) || read_all(f, p0, (size_t)n * 4) ||
        read_all(f, grads, (size_t)(K * n) * 2))
        return 1;
    fclose(f);

    /* device state: fp32 master/m/v, bf16 weights and gradients */
    float *d_p, *d_m, *d_v;
    uint16_t *d_w, *d_g;
    void *d_ring, *d_ws;
    const size_t ring_bytes = 1 << 20;
    const size_t ws_bytes = gockpt_workspace_bytes(n);
    CHECK_HIP(hipMalloc((void**)&d_p, (size_t)n * 4));
    CHECK_HIP(hipMalloc((void**)&d_m, (size_t)n * 4));
    CHECK_HIP(hipMalloc((void**)&d_v, (size_t)n * 4));
    CHECK_HIP(hipMalloc((void**)&d_w, (size_t)n * 2));
    CHECK_HIP(hipMalloc((void**)&d_g, (size_t)n * 2));
    CHECK_HIP(hipMalloc(&d_ring, ring_bytes));
    CHECK_HIP(hipMalloc(&d_ws, ws_bytes));
    CHECK_HIP(hipMemcpy(d_p, p0, (size_t)n * 4, hipMemcpyHostToDevice));
    CHECK_HIP(hipMemset(d_m, 0, (size_t)n * 4));
    CHECK_HIP(hipMemset(d_v, 0, (size_t)n * 4));
    hipStream_t cs, xs;
    CHECK_HIP(hipStreamCreateWithFlags(&cs, hipStreamNonBlocking));
    CHECK_HIP(hipStreamCreateWithFlags(&xs, hipStreamNonBlocking));

    gockpt_config cfg;
    memset(&cfg, 0, sizeof cfg);
    cfg.n = n;
    cfg.master = d_p;
    cfg.exp_avg = d_m;
    cfg.exp_avg_sq = d_v;
    cfg.weight_bf16 = d_w;
    cfg.grad16 = d_g;
    cfg.beta1 = 0.9;
    cfg.beta2 = 0.999;
    cfg.eps = 1e-8;
    cfg.weight_decay = 0.01;
    cfg.check_overflow = 1;
    cfg.dynamic_scale = 0;
    cfg.init_scale = 1.0f;
    cfg.growth_factor = 2.0f;
    cfg.backoff_factor = 0.5f;
    cfg.min_scale = 1.0f;
    cfg.growth_interval = 1000;
    cfg.ring = d_ring;
    cfg.ring_bytes = ring_bytes;
    cfg.copy_bytes = 64 << 10;
    cfg.workspace = d_ws;
    cfg.workspace_bytes = ws_bytes;
    cfg.compute_stream = cs;
    cfg.copy_stream = xs;
    cfg.grad_dtype = GOCKPT_GRAD_BF16;

    gockpt_ctx* ctx = NULL;
    CHECK_G(NULL, gockpt_create(&cfg, &ctx));

    gockpt_arena_layout lay;
    CHECK_G(ctx, gockpt_arena_layout_for((int)K, bounds, n, &lay, NULL));
    void* arena = NULL;
    CHECK_G(NULL, gockpt_host_alloc(lay.total, &arena));
    /* the ring plan that never blocks the caller, and each step's copies
       queued at the next call into the library */
    gockpt_window_opts opts;
    memset(&opts, 0, sizeof opts);
    opts.late_plan = GOCKPT_RING_DEVICE_WAIT;
    opts.defer_copies = 1;
    CHECK_G(ctx, gockpt_begin_window_ex(ctx, (int)K, bounds, arena, lay.total, &opts));
    for (int64_t s = 0; s < K; ++s) {
        CHECK_G(ctx, gockpt_backward_begin(ctx, NULL));
        CHECK_HIP(hipMemcpyAsync(d_g, grads + s * n, (size_t)n * 2, hipMemcpyHostToDevice, cs));
        CHECK_G(ctx, gockpt_step(ctx, 1e-4f));
    }
    gockpt_window_stats stats;
    CHECK_G(ctx, gockpt_drain(ctx, 1, &stats));

    float* out_p = malloc((size_t)n * 4);
    float* out_m = malloc((size_t)n * 4);
    float* out_v = malloc((size_t)n * 4);
    uint16_t* out_w = malloc((size_t)n * 2);
    float* dev_p = malloc((size_t)n * 4);
    if (!out_p || !out_m || !out_v || !out_w || !dev_p) return 1;
    gockpt_ckpt_meta meta;
    /* the replay in a library thread, then the wait (the blocking form,
       gockpt_restore, takes the same arguments plus &meta) */
    CHECK_G(ctx, gockpt_restore_async(ctx, out_p, out_m, out_v, out_w, 4));
    CHECK_G(ctx, gockpt_restore_wait(ctx, &meta));
    CHECK_HIP(hipStreamSynchronize(cs));
    CHECK_HIP(hipMemcpy(dev_p, d_p, (size_t)n * 4, hipMemcpyDeviceToHost));

    FILE* o = fopen(argv[2], "wb");
    if (!o) return 1;
    int64_t t = meta.t;
    fwrite(out_p, 4, (size_t)n, o);
    fwrite(out_m, 4, (size_t)n, o);
    fwrite(out_v, 4, (size_t)n, o);
    fwrite(out_w, 2, (size_t)n, o);
    fwrite(dev_p, 4, (size_t)n, o);
    fwrite(&t, 8, 1, o);
    fclose(o);

    CHECK_G(ctx, gockpt_destroy(ctx));
    CHECK_G(NULL, gockpt_host_free(arena));
    hipFree(d_p);
    hipFree(d_m);
    hipFree(d_v);
    hipFree(d_w);
    hipFree(d_g);
    hipFree(d_ring);
    hipFree(d_ws);
    hipStreamDestroy(cs);
    hipStreamDestroy(xs);
    printf("window_c: n=%lld K=%lld t=%lld copies=%.0f bytes\n", (long long)n, (long long)K, (long long)t,
           (double)stats.bytes_d2h);
    return 0;
}
