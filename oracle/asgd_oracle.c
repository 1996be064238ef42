/*
 * Plain CPU oracle of the ASGD parameter-server update (test infrastructure).
 *
 * This file is test infrastructure: only the tests, the smoke check and the
 * CPU-baseline leg of the benchmark load it. It shares no code with the GPU
 * library and is deliberately slow and simple: one loop over the coordinates
 * per pushed gradient, in the order the paper states the update.
 *
 * Build: C99, -O2 -ffp-contract=off, no fast-math, x86-64 SSE scalar binary32
 * arithmetic with round-to-nearest-even and no flush-to-zero. Every product
 * and every difference below is rounded to float on its own.
 *
 * Precision: the paper stores weights and gradients as 32-bit floats (Sec. 4.4,
 * "Half-precision floating point operations"), so each step computes in
 * binary32; lr and momentum arrive as C floats.
 *
 * Pins (tests/test_oracle_pins.py): closed forms of the constant-gradient
 * run, zero gradients, an exact-rational evaluation with round-to-nearest-even
 * after every operation over every arrival order of small cases, and torch's
 * bfloat16 conversions. The momentum step is pinned to its own closed form
 * only: the paper has no momentum, so against the paper it is parity
 * unpinned.
 */
#include <stddef.h>
#include <stdint.h>
#include <string.h>

/* One SGD step on every coordinate k (Eq. "gd", Sec. 2.1):
 *   theta_k <- theta_k - alpha * grad_k
 * ASGD (Eq. "asgd") applies it once per gradient received, with the gradient
 * of whichever learner sent it. Rounding: p = fl(alpha * g), w = fl(w - p). */
void orc_step_f32(float *w, const float *g, size_t n, float lr)
{
    for (size_t i = 0; i < n; ++i) {
        float p = lr * g[i];
        w[i] = w[i] - p;
    }
}

/* The same step with heavy-ball momentum kept by the server, one step per
 * push (the paper has no momentum; this is the Torch SGD convention with no
 * dampening and no Nesterov term):
 *   v_k <- m * v_k + g_k ;  theta_k <- theta_k - alpha * v_k
 * Rounding: t = fl(m*v), v = fl(t + g), p = fl(alpha*v), w = fl(w - p). */
void orc_step_mom_f32(float *w, float *v, const float *g, size_t n, float lr, float m)
{
    for (size_t i = 0; i < n; ++i) {
        float t = m * v[i];
        v[i] = t + g[i];
        float p = lr * v[i];
        w[i] = w[i] - p;
    }
}

/* bfloat16 -> binary32: a bf16 value is the upper 16 bits of a binary32 with
 * the lower 16 bits zero, so the widening is exact. */
float orc_bf16_to_f32(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

/* Widen a whole bf16 buffer (used to check the widening bit for bit). */
void orc_widen_bf16(float *dst, const uint16_t *src, size_t n)
{
    for (size_t i = 0; i < n; ++i)
        dst[i] = orc_bf16_to_f32(src[i]);
}

/* binary32 -> bfloat16, round to nearest, ties to even, written from the
 * definition: keep the upper 16 bits; the discarded lower 16 bits decide.
 * Above half an ulp rounds up, below rounds down, exactly half rounds to the
 * candidate with an even last bit. A carry out of the mantissa moves to the
 * next binade (and to infinity past the largest finite value), which is the
 * correct rounded result. NaN stays NaN (quiet bit set, sign kept). */
uint16_t orc_f32_to_bf16(float f)
{
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu) != 0)
        return (uint16_t)((u >> 16) | 0x0040u);
    uint32_t hi = u >> 16;
    uint32_t lo = u & 0xffffu;
    if (lo > 0x8000u)
        hi += 1;
    else if (lo == 0x8000u && (hi & 1u))
        hi += 1;
    return (uint16_t)hi;
}

/* ASGD step with a bf16 gradient and fp32 master weights: the gradient is
 * widened (exactly) and the fp32 step above is taken. */
void orc_step_bf16(float *w, const uint16_t *g, size_t n, float lr)
{
    for (size_t i = 0; i < n; ++i) {
        float x = orc_bf16_to_f32(g[i]);
        float p = lr * x;
        w[i] = w[i] - p;
    }
}

void orc_step_mom_bf16(float *w, float *v, const uint16_t *g, size_t n, float lr, float m)
{
    for (size_t i = 0; i < n; ++i) {
        float x = orc_bf16_to_f32(g[i]);
        float t = m * v[i];
        v[i] = t + x;
        float p = lr * v[i];
        w[i] = w[i] - p;
    }
}

/* A pull: the learner's weight buffer receives the server's weights
 * (Sec. 4.1, the weights staging buffer), as fp32 or rounded to bf16. */
void orc_pull_f32(float *dst, const float *w, size_t n)
{
    for (size_t i = 0; i < n; ++i)
        dst[i] = w[i];
}

void orc_pull_bf16(uint16_t *dst, const float *w, size_t n)
{
    for (size_t i = 0; i < n; ++i)
        dst[i] = orc_f32_to_bf16(w[i]);
}

/* Synchronous SGD step (Eq. "ssgd", Sec. 2.1): the server averages the
 * lambda gradients it collected, one per learner, and takes one step of
 * Eq. "gd" with the average. The sum runs in learner order 1..lambda from
 * +0, then is divided by lambda (correctly rounded division), then the step.
 * grads points at lambda gradient pointers of n values; is_bf16 says they hold
 * bf16 bit patterns. With v non-NULL the heavy-ball form is used with the
 * average as the gradient. */
void orc_ssgd_step(float *w, float *v, const void *const *grads, int lambda, int is_bf16,
                   size_t n, float lr, float m)
{
    for (size_t i = 0; i < n; ++i) {
        float s = 0.0f;
        for (int l = 0; l < lambda; ++l) {
            float x = is_bf16 ? orc_bf16_to_f32(((const uint16_t *)grads[l])[i])
                              : ((const float *)grads[l])[i];
            s = s + x;
        }
        float avg = s / (float)lambda;
        if (v != NULL) {
            float t = m * v[i];
            v[i] = t + avg;
            float p = lr * v[i];
            w[i] = w[i] - p;
        } else {
            float p = lr * avg;
            w[i] = w[i] - p;
        }
    }
}
