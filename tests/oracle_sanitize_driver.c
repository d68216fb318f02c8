/* Drives every function of the CPU oracle (oracle/monomoe_oracle.c) over small inputs and
 * edge cases, for a build with AddressSanitizer and UndefinedBehaviorSanitizer: any
 * out-of-bounds access, use of uninitialised heap through ASan's checks, signed overflow,
 * bad shift or misaligned access aborts the run.  The checks below are light invariants;
 * the numerical pins live in the Python oracle tests.  Prints "ok" and exits 0 on success. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "monomoe_oracle.h"

static uint64_t rng = 0x9E3779B97F4A7C15ull;
static uint32_t next_u32(void) {   /* xorshift64* */
    rng ^= rng >> 12;
    rng ^= rng << 25;
    rng ^= rng >> 27;
    return (uint32_t)((rng * 0x2545F4914F6CDD1Dull) >> 32);
}
static float uniform(float a) { return a * ((float)next_u32() / 4294967296.0f * 2.0f - 1.0f); }
static uint16_t bf16_of(float f) {   /* truncation is enough for test data */
    uint32_t u;
    memcpy(&u, &f, 4);
    return (uint16_t)(u >> 16);
}

#define CHECK(c)                                                       \
    do {                                                               \
        if (!(c)) {                                                    \
            fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
            return 1;                                                  \
        }                                                              \
    } while (0)

static int codec(void) {
    for (int c = 0; c < 256; ++c) {
        const double v = mo_e4m3_decode((uint8_t)c);
        if (isnan(v)) continue;
        CHECK(mo_e4m3_encode((float)v) == (uint8_t)c);
    }
    CHECK(mo_e4m3_encode(NAN) == 0x7F);
    CHECK(mo_e4m3_encode(1e30f) == 0x7E && mo_e4m3_encode(-1e30f) == 0xFE);
    for (uint32_t b = 0; b < 65536; ++b) (void)mo_bf16_decode((uint16_t)b);
    float v[128], s;
    uint8_t q[128];
    memset(v, 0, sizeof v);
    mo_quantize_group(v, 128, q, &s);
    CHECK(s == 0.0f);
    for (int i = 0; i < 128; ++i) CHECK(q[i] == 0);
    for (int i = 0; i < 128; ++i) v[i] = uniform(3.0f);
    v[17] = -1e6f;
    mo_quantize_group(v, 128, q, &s);
    CHECK(s > 0.0f && fabs(mo_e4m3_decode(q[17]) * s + 1e6) <= 1e6 * 0.0625);
    for (int i = 0; i < 128; ++i) v[i] = 1e-42f;   /* subnormal group */
    mo_quantize_group(v, 128, q, &s);
    return 0;
}

static int routing(void) {
    enum { T = 3, E = 8 };
    double logits[T * E], w[T * E];
    int32_t ids[T * E];
    float sel[E];
    for (int i = 0; i < T * E; ++i) logits[i] = uniform(4.0f);
    logits[5] = logits[6];   /* an exact tie */
    for (int e = 0; e < E; ++e) sel[e] = uniform(0.1f);
    for (int renorm = 0; renorm < 2; ++renorm) {
        for (int k = 1; k <= E; ++k) {
            mo_select(T, E, k, renorm, logits, ids, w);
            for (int i = 0; i < T * k; ++i) CHECK(ids[i] >= 0 && ids[i] < E && w[i] >= 0.0);
            mo_select_sigmoid(T, E, k, logits, renorm ? sel : NULL, 2.5, ids, w);
            for (int i = 0; i < T * k; ++i) CHECK(ids[i] >= 0 && ids[i] < E && w[i] >= 0.0);
        }
    }
    return 0;
}

static int forward(void) {
    enum { T = 3, H = 256, E = 8, I = 256, K = 2 };
    uint16_t* x = malloc(sizeof(uint16_t) * T * H);
    uint16_t* rw = malloc(sizeof(uint16_t) * E * H);
    float* bias = malloc(sizeof(float) * E);
    uint8_t* w13[E];
    float* w13s[E];
    uint8_t* w2[E];
    float* w2s[E];
    for (int i = 0; i < T * H; ++i) x[i] = bf16_of(uniform(1.0f));
    for (int i = 0; i < H; ++i) x[H + i] = 0;   /* token 1: all zero */
    for (int i = 0; i < E * H; ++i) rw[i] = bf16_of(uniform(0.05f));
    for (int e = 0; e < E; ++e) bias[e] = uniform(0.5f);
    for (int e = 0; e < E; ++e) {
        w13[e] = malloc((size_t)2 * I * H);
        w13s[e] = malloc(sizeof(float) * (2 * I / 128) * (H / 128));
        w2[e] = malloc((size_t)H * I);
        w2s[e] = malloc(sizeof(float) * (H / 128) * (I / 128));
        for (int i = 0; i < 2 * I * H; ++i) w13[e][i] = (uint8_t)(next_u32() & 0xFF) & 0xF7;  /* no NaN codes */
        for (int i = 0; i < H * I; ++i) w2[e][i] = (uint8_t)(next_u32() & 0xFF) & 0xF7;
        for (int i = 0; i < (2 * I / 128) * (H / 128); ++i) w13s[e][i] = 1e-3f;
        for (int i = 0; i < (H / 128) * (I / 128); ++i) w2s[e][i] = e == 3 ? 0.0f : 1e-3f;   /* a zero-scale expert */
    }
    double* ref = malloc(sizeof(double) * T * H);
    mo_debug_t d;
    d.ids = malloc(sizeof(int32_t) * T * K);
    d.w = malloc(sizeof(double) * T * K);
    d.xq = malloc((size_t)T * H);
    d.xs = malloc(sizeof(float) * T * (H / 128));
    d.h = malloc(sizeof(double) * T * K * 2 * I);
    d.act = malloc(sizeof(double) * T * K * I);
    d.aq = malloc((size_t)T * K * I);
    d.as = malloc(sizeof(float) * T * K * (I / 128));
    d.y = malloc(sizeof(double) * T * K * H);
    CHECK(mo_forward(T, H, E, I, K, 1, x, rw, bias, (const uint8_t* const*)w13, (const float* const*)w13s,
                     (const uint8_t* const*)w2, (const float* const*)w2s, NULL, NULL, ref, &d) == 0);
    for (int i = 0; i < T * H; ++i) CHECK(isfinite(ref[i]));
    for (int i = 0; i < H; ++i) CHECK(ref[H + i] == 0.0);   /* the zero token */
    CHECK(mo_forward_policy(T, H, E, I, K, 0, MO_ROUTING_SIGMOID_BIAS, bias, 2.5, x, rw, NULL,
                            (const uint8_t* const*)w13, (const float* const*)w13s, (const uint8_t* const*)w2,
                            (const float* const*)w2s, NULL, NULL, ref, NULL) == 0);
    const int32_t inj[T * K] = {3, 0, 1, 2, 7, 6};
    const double injw[T * K] = {0.5, 0.5, 1.0, 0.0, 0.25, 0.75};
    CHECK(mo_forward(T, H, E, I, K, 1, x, rw, NULL, (const uint8_t* const*)w13, (const float* const*)w13s,
                     (const uint8_t* const*)w2, (const float* const*)w2s, inj, injw, ref, &d) == 0);
    /* refusals: a shape off the 128 grid, k out of range, a selected expert without weights */
    CHECK(mo_forward(T, 200, E, I, K, 1, x, rw, NULL, (const uint8_t* const*)w13, (const float* const*)w13s,
                     (const uint8_t* const*)w2, (const float* const*)w2s, NULL, NULL, ref, NULL) == -1);
    CHECK(mo_forward(T, H, E, I, 0, 1, x, rw, NULL, (const uint8_t* const*)w13, (const float* const*)w13s,
                     (const uint8_t* const*)w2, (const float* const*)w2s, NULL, NULL, ref, NULL) == -1);
    uint8_t* saved = w13[3];
    w13[3] = NULL;
    CHECK(mo_forward(T, H, E, I, K, 1, x, rw, NULL, (const uint8_t* const*)w13, (const float* const*)w13s,
                     (const uint8_t* const*)w2, (const float* const*)w2s, inj, injw, ref, NULL) == -1);
    w13[3] = saved;
    for (int e = 0; e < E; ++e) {
        free(w13[e]);
        free(w13s[e]);
        free(w2[e]);
        free(w2s[e]);
    }
    free(d.ids); free(d.w); free(d.xq); free(d.xs); free(d.h); free(d.act); free(d.aq); free(d.as); free(d.y);
    free(ref);
    free(x);
    free(rw);
    free(bias);
    return 0;
}

int main(void) {
    if (codec() || routing() || forward()) return 1;
    printf("ok\n");
    return 0;
}
