/* Drives every function of the C oracle on small and edge-sized inputs so
 * that AddressSanitizer / UndefinedBehaviorSanitizer can check them (built
 * and run by tests/test_sanitizers.py on the host). Exit status 0 = no
 * finding; the sanitizers abort on the first one. */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

void orc_step_f32(float *w, const float *g, size_t n, float lr);
void orc_step_mom_f32(float *w, float *v, const float *g, size_t n, float lr, float m);
float orc_bf16_to_f32(uint16_t b);
void orc_widen_bf16(float *dst, const uint16_t *src, size_t n);
uint16_t orc_f32_to_bf16(float f);
void orc_step_bf16(float *w, const uint16_t *g, size_t n, float lr);
void orc_step_mom_bf16(float *w, float *v, const uint16_t *g, size_t n, float lr, float m);
void orc_pull_f32(float *dst, const float *w, size_t n);
void orc_pull_bf16(uint16_t *dst, const float *w, size_t n);
void orc_ssgd_step(float *w, float *v, const void *const *grads, int lambda, int is_bf16,
                   size_t n, float lr, float m);

static float *falloc(size_t n, float x)
{
    float *p = malloc((n ? n : 1) * sizeof *p); /* exact sizes: overruns are caught */
    for (size_t i = 0; i < n; ++i)
        p[i] = x * (float)(i % 7) - 0.01f;
    return p;
}

int main(void)
{
    const size_t sizes[] = {0, 1, 2, 7, 64, 1001};
    for (size_t s = 0; s < sizeof sizes / sizeof sizes[0]; ++s) {
        size_t n = sizes[s];
        float *w = falloc(n, 0.01f), *v = falloc(n, 0.0f), *g = falloc(n, 0.001f);
        float *d = falloc(n, 0.0f);
        uint16_t *gb = malloc((n ? n : 1) * sizeof *gb), *db = malloc((n ? n : 1) * sizeof *db);
        for (size_t i = 0; i < n; ++i)
            gb[i] = orc_f32_to_bf16(g[i]);
        orc_step_f32(w, g, n, 0.01f);
        orc_step_mom_f32(w, v, g, n, 0.01f, 0.9f);
        orc_step_bf16(w, gb, n, 0.01f);
        orc_step_mom_bf16(w, v, gb, n, 0.01f, 0.9f);
        orc_pull_f32(d, w, n);
        orc_pull_bf16(db, w, n);
        orc_widen_bf16(d, db, n);
        for (int lambda = 1; lambda <= 9; lambda += 4) {
            const void **gs = malloc((size_t)lambda * sizeof *gs);
            for (int l = 0; l < lambda; ++l)
                gs[l] = g;
            orc_ssgd_step(w, v, gs, lambda, 0, n, 0.01f, 0.9f);
            orc_ssgd_step(w, NULL, gs, lambda, 0, n, 0.01f, 0.0f);
            for (int l = 0; l < lambda; ++l)
                gs[l] = gb;
            orc_ssgd_step(w, v, gs, lambda, 1, n, 0.01f, 0.9f);
            free(gs);
        }
        for (size_t i = 0; i < n; ++i)
            if (!isfinite(w[i]))
                return 2;
        free(w); free(v); free(g); free(d); free(gb); free(db);
    }
    /* every bf16 pattern and the fp32 specials through the conversions */
    for (uint32_t b = 0; b < 65536; ++b) {
        float f = orc_bf16_to_f32((uint16_t)b);
        (void)orc_f32_to_bf16(f);
    }
    const float specials[] = {0.0f, -0.0f, INFINITY, -INFINITY, NAN, 3.4028235e38f, 1e-45f};
    for (size_t i = 0; i < sizeof specials / sizeof specials[0]; ++i)
        (void)orc_f32_to_bf16(specials[i]);
    puts("sanitized run clean");
    return 0;
}
