/*
 * The C ABI from plain C: no Python, no torch. Device memory comes from the
 * HIP runtime directly. Checked against closed forms that hold exactly in
 * binary32 (dyadic values, so every product and difference is exact):
 *
 *   - constant gradient g, no momentum, T pushes: w_T = w_0 - T*lr*g
 *     (Eq. "gd" applied T times);
 *   - momentum m = 1/2, T pushes from v_0 = 0: v_T = g*(1 - m^T)/(1 - m),
 *     w_T = w_0 - lr*g/(1 - m) * (T - m*(1 - m^T)/(1 - m));
 *
 * plus the queue contract (a full queue refuses the push, Sec. 4.1), the
 * timestamp (one per applied gradient, Sec. 2.1), a bf16 pull (w rounded to
 * nearest even) and server-owned rows. Then times 20,000 Tiny-shaped
 * push + apply_pull steps (no Python in the loop). Built by the package
 * build next to the library and run by tests/test_c_abi.py on a GPU.
 * Prints "c abi ok".
 */
#define _POSIX_C_SOURCE 199309L
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>
#include <time.h>

#include "ps.h"

#define CHECK(cond, ...)                                                   \
    do {                                                                   \
        if (!(cond)) {                                                     \
            fprintf(stderr, "c_abi_smoke: " __VA_ARGS__);                  \
            fprintf(stderr, " (last error: %s)\n", ps_last_error());       \
            exit(1);                                                       \
        }                                                                  \
    } while (0)

#define HIPCHECK(x)                                                        \
    do {                                                                   \
        hipError_t e_ = (x);                                               \
        CHECK(e_ == hipSuccess, "%s: %s", #x, hipGetErrorString(e_));      \
    } while (0)

static float *fill_device(size_t n, float value)
{
    float *h = malloc(n * sizeof *h);
    float *d = NULL;
    CHECK(h != NULL, "host allocation");
    for (size_t i = 0; i < n; ++i) h[i] = value;
    HIPCHECK(hipMalloc((void **)&d, n * sizeof *d));
    HIPCHECK(hipMemcpy(d, h, n * sizeof *d, hipMemcpyHostToDevice));
    free(h);
    return d;
}

static void expect_all(const float *dev, size_t n, float want, const char *what)
{
    float *h = malloc(n * sizeof *h);
    CHECK(h != NULL, "host allocation");
    HIPCHECK(hipMemcpy(h, dev, n * sizeof *h, hipMemcpyDeviceToHost));
    for (size_t i = 0; i < n; ++i) {
        uint32_t a, b;
        memcpy(&a, &h[i], 4);
        memcpy(&b, &want, 4);
        CHECK(a == b, "%s[%zu] = %.9g, want %.9g", what, i, h[i], want);
    }
    free(h);
}

int main(void)
{
    const size_t n = (size_t)1 << 20 | 3;    /* vector path plus a ragged tail */
    const float lr = 1.0f / 128, g = 1.0f / 1024, w0 = 1.0f;
    int count = 0;
    if (hipGetDeviceCount(&count) != hipSuccess || count < 1) {
        fprintf(stderr, "c_abi_smoke: no GPU\n");
        return 2;
    }

    /* no momentum: 40 pushes, depth 32, so a full queue and two applies */
    ps_server *ps = ps_create(n, lr, 0.0f);
    CHECK(ps != NULL, "ps_create");
    CHECK(ps_velocity(ps) == NULL, "no velocity without momentum");
    float *w_init = fill_device(n, w0);
    float *grad = fill_device(n, g);
    CHECK(ps_set_weights(ps, w_init) == PS_OK, "ps_set_weights");
    CHECK(ps_set_queue_depth(ps, 32) == PS_OK, "ps_set_queue_depth");
    int pushed = 0;
    for (int j = 0; j < 40; ++j) {
        int rc = ps_push(ps, j % 5, grad);
        if (rc == PS_EFULL) {
            CHECK(pushed == 32 && ps_pending(ps) == 32, "EFULL only on a full queue");
            CHECK(ps_apply_pending(ps) == PS_OK, "ps_apply_pending");
            rc = ps_push(ps, j % 5, grad);
        }
        CHECK(rc == PS_OK, "ps_push %d", j);
        ++pushed;
    }
    CHECK(ps_apply_pending(ps) == PS_OK, "second ps_apply_pending");
    CHECK(ps_timestamp(ps) == 40, "timestamp %llu, want 40",
          (unsigned long long)ps_timestamp(ps));
    float *rep = NULL;
    uint16_t *rep16 = NULL;
    HIPCHECK(hipMalloc((void **)&rep, n * sizeof *rep));
    HIPCHECK(hipMalloc((void **)&rep16, n * sizeof *rep16));
    CHECK(ps_pull(ps, 0, rep) == PS_OK, "ps_pull");
    int ids[1] = {1};
    void *dsts[1] = {rep16};
    CHECK(ps_pull_many(ps, 1, ids, dsts, PS_BF16) == PS_OK, "ps_pull_many bf16");
    CHECK(ps_sync(ps) == PS_OK, "ps_sync");
    const float want = w0 - 40.0f * (lr * g);    /* exact: all terms dyadic */
    expect_all(ps_weights(ps), n, want, "w (no momentum)");
    expect_all(rep, n, want, "fp32 replica");
    {
        uint16_t *h = malloc(n * sizeof *h);
        CHECK(h != NULL, "host allocation");
        HIPCHECK(hipMemcpy(h, rep16, n * sizeof *h, hipMemcpyDeviceToHost));
        /* 1 - 40 * 2^-17 lies within 2^-9 of 1.0, so it rounds to bf16 1.0 */
        for (size_t i = 0; i < n; ++i) CHECK(h[i] == 0x3F80, "bf16 replica[%zu] = %04x", i, h[i]);
        free(h);
    }
    ps_stats st;
    CHECK(ps_get_stats(ps, &st) == PS_OK, "ps_get_stats");
    CHECK(st.pushes_accepted == 40 && st.pushes_rejected == 1 && st.applies == 2 &&
              st.pushes_applied == 40,
          "stats: accepted %llu rejected %llu applies %llu applied %llu",
          (unsigned long long)st.pushes_accepted, (unsigned long long)st.pushes_rejected,
          (unsigned long long)st.applies, (unsigned long long)st.pushes_applied);
    ps_destroy(ps);

    /* momentum 1/2, 8 pushes, gradients in server-owned rows */
    const float m = 0.5f;
    ps = ps_create(n, lr, m);
    CHECK(ps != NULL, "ps_create with momentum");
    CHECK(ps_set_weights(ps, w_init) == PS_OK, "ps_set_weights");
    void *rows[8];
    CHECK(ps_alloc_rows(ps, 8, PS_F32, rows) == PS_OK, "ps_alloc_rows");
    for (int j = 0; j < 8; ++j) {
        /* rows of 2 MiB or more sit at phase ((j + 2) * 1.75 MiB) mod 2 MiB */
        CHECK(((uintptr_t)rows[j] % ((uintptr_t)2 << 20)) ==
                  ((uintptr_t)(j + 2) * ((uintptr_t)7 << 18)) % ((uintptr_t)2 << 20),
              "row %d phase", j);
        HIPCHECK(hipMemcpy(rows[j], grad, n * sizeof(float), hipMemcpyDeviceToDevice));
        CHECK(ps_push(ps, j, rows[j]) == PS_OK, "push row %d", j);
    }
    CHECK(ps_free_rows(ps, rows[0]) == PS_ESTATE, "rows with pending gradients are kept");
    CHECK(ps_apply_pending(ps) == PS_OK, "momentum apply");
    CHECK(ps_sync(ps) == PS_OK, "ps_sync");
    const int T = 8;
    double mt = 1.0;
    for (int t = 0; t < T; ++t) mt *= m;
    const double v_want = g * (1.0 - mt) / (1.0 - m);
    const double w_want = w0 - lr * g / (1.0 - m) * (T - m * (1.0 - mt) / (1.0 - m));
    expect_all(ps_velocity(ps), n, (float)v_want, "v (momentum 1/2)");
    expect_all(ps_weights(ps), n, (float)w_want, "w (momentum 1/2)");
    CHECK((double)(float)v_want == v_want && (double)(float)w_want == w_want,
          "closed forms exact in binary32");
    CHECK(ps_free_rows(ps, rows[0]) == PS_OK, "ps_free_rows");
    CHECK(ps_free_rows(ps, rows[0]) == PS_EINVAL, "second ps_free_rows");
    ps_destroy(ps);

    /* the Tiny shape (2^20 parameters, one gradient per apply, the pushing
     * learner pulls after every push) driven from C: the library's own cost
     * per push, with no Python in the loop; gradients cycle over 8 rows */
    {
        const size_t nt = (size_t)1 << 20;
        ps = ps_create(nt, 0.01f, 0.0f);
        CHECK(ps != NULL, "ps_create (tiny)");
        CHECK(ps_set_queue_depth(ps, 1) == PS_OK, "depth 1");
        void *g8[8];
        CHECK(ps_alloc_rows(ps, 8, PS_F32, g8) == PS_OK, "rows (tiny)");
        for (int j = 0; j < 8; ++j) HIPCHECK(hipMemset(g8[j], 0, nt * sizeof(float)));
        void *d = rep;
        const int steps = 20000;
        struct timespec t0, t1;
        CHECK(ps_sync(ps) == PS_OK, "sync");
        clock_gettime(CLOCK_MONOTONIC, &t0);
        for (int j = 0; j < steps; ++j) {
            int l = j & 3;
            CHECK(ps_push(ps, l, g8[j & 7]) == PS_OK, "tiny push");
            CHECK(ps_apply_pull(ps, 1, &l, &d, PS_F32) == PS_OK, "tiny apply_pull");
        }
        CHECK(ps_sync(ps) == PS_OK, "sync");
        clock_gettime(CLOCK_MONOTONIC, &t1);
        const double s = (double)(t1.tv_sec - t0.tv_sec) + 1e-9 * (double)(t1.tv_nsec - t0.tv_nsec);
        CHECK(ps_timestamp(ps) == (uint64_t)steps, "tiny timestamp");
        printf("tiny loop: %.2f us per push+apply+pull, %.0f pushes/s\n", s / steps * 1e6, steps / s);
        ps_destroy(ps);
    }

    HIPCHECK(hipFree(w_init));
    HIPCHECK(hipFree(grad));
    HIPCHECK(hipFree(rep));
    HIPCHECK(hipFree(rep16));
    printf("c abi ok\n");
    return 0;
}
