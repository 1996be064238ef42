/*
 * A CPU parameter server in the paper's own style (test infrastructure).
 *
 * This file is test infrastructure: only the tests and the CPU-baseline leg
 * of the benchmark load it, as context beside the oracle. It shares no code
 * with the GPU library.
 *
 * The paper's server keeps the weights in host shared memory and applies
 * each received gradient as one pass over them with a few OpenMP threads,
 * the vector loop unrolled eight times (Sec. 4.1; Sec. 4.4 reports the
 * unrolled loop 30% faster than a plain one and a 16-bit software path 5x
 * slower). Here: one pass per gradient, in arrival order, the coordinates
 * split over `threads` OpenMP threads, eight coordinates per loop iteration.
 * Each coordinate still sees the gradients one after another with the same
 * roundings as the oracle (no contraction), so results are bitwise equal to
 * the oracle's; tests/test_cpu_ps.py checks that.
 */
#include <stddef.h>
#include <stdint.h>
#include <string.h>

static float widen(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

/* One gradient over w (and v): the step of Eq. "gd" per coordinate, or its
 * heavy-ball form; is_bf16 selects 16-bit gradients widened exactly. */
void cps_step(float *w, float *v, const void *grad, int is_bf16, size_t n, float lr, float m,
              int threads)
{
    const float *g32 = (const float *)grad;
    const uint16_t *g16 = (const uint16_t *)grad;
    const size_t n8 = n / 8 * 8;
    #pragma omp parallel num_threads(threads)
    {
        #pragma omp for schedule(static)
        for (size_t i = 0; i < n8; i += 8) {
            float g[8];
            for (int e = 0; e < 8; ++e)
                g[e] = is_bf16 ? widen(g16[i + e]) : g32[i + e];
            if (v) {
                for (int e = 0; e < 8; ++e) {
                    float t = m * v[i + e];
                    v[i + e] = t + g[e];
                    float p = lr * v[i + e];
                    w[i + e] = w[i + e] - p;
                }
            } else {
                for (int e = 0; e < 8; ++e) {
                    float p = lr * g[e];
                    w[i + e] = w[i + e] - p;
                }
            }
        }
    }
    for (size_t i = n8; i < n; ++i) {
        float x = is_bf16 ? widen(g16[i]) : g32[i];
        if (v) {
            float t = m * v[i];
            v[i] = t + x;
            float p = lr * v[i];
            w[i] = w[i] - p;
        } else {
            float p = lr * x;
            w[i] = w[i] - p;
        }
    }
}

/* A pull: copy w into a replica with `threads` threads. */
void cps_pull(float *dst, const float *w, size_t n, int threads)
{
    const size_t chunk = 1u << 16;
    #pragma omp parallel for num_threads(threads) schedule(static)
    for (size_t i = 0; i < n; i += chunk)
        memcpy(dst + i, w + i, (n - i < chunk ? n - i : chunk) * sizeof(float));
}
