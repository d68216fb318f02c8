/*
 * monomoe_oracle.c -- plain fp64 CPU oracle of the routed-MoE decode operator of
 * MonoMoE (arXiv 2609.04244).  TEST INFRASTRUCTURE ONLY: see monomoe_oracle.h.
 *
 * Written for a reader checking it against the paper by eye: one loop nest per step,
 * token-major, no blocking, no fusion, no reordering beyond the definitions.
 */
#include "monomoe_oracle.h"

#include <float.h>
#include <math.h>
#include <stdlib.h>
#include <string.h>

/* The quantiser's two fp32 operations must be evaluated in fp32, not in a wider type. */
#if !defined(FLT_EVAL_METHOD) || FLT_EVAL_METHOD != 0
#error "the oracle needs FLT_EVAL_METHOD == 0 (fp32 arithmetic evaluated in fp32)"
#endif

/* ---------------------------------------------------------------------------------
 * E4M3FN codec (the E4M3 format named in Sec. 4.1; OCP 8-bit floating point spec).
 * value = (-1)^s * 2^(e-7) * (1 + m/8)   for exponent field e in 1..15
 *       = (-1)^s * 2^(-6)  * (m/8)       for e == 0 (subnormal)
 * e == 15 with m == 7 is NaN; there is no infinity.
 * ------------------------------------------------------------------------------- */
double mo_e4m3_decode(uint8_t code)
{
    int s = (code >> 7) & 1;
    int e = (code >> 3) & 15;
    int m = code & 7;
    double mag;
    if (e == 15 && m == 7) return NAN;
    if (e == 0) mag = ldexp((double)m / 8.0, -6);
    else        mag = ldexp(1.0 + (double)m / 8.0, e - 7);
    return s ? -mag : mag;
}

/* Round y >= 0 to the nearest integer, ties to the even integer.  Exact for the
 * doubles this file produces (small integers plus a binary fraction). */
static double round_half_even(double y)
{
    double f = floor(y);
    double d = y - f;
    if (d > 0.5) return f + 1.0;
    if (d < 0.5) return f;
    return (fmod(f, 2.0) == 0.0) ? f : f + 1.0;
}

uint8_t mo_e4m3_encode(float v)
{
    uint8_t sign;
    double a;
    if (isnan(v)) return 0x7F;
    sign = signbit(v) ? 0x80 : 0x00;
    a = fabs((double)v);
    if (a >= 448.0) return (uint8_t)(sign | 0x7E);           /* saturate */
    if (a < ldexp(1.0, -6)) {
        /* subnormal range: step 2^-9; m == 8 lands on the smallest normal, code 0x08 */
        double m = round_half_even(a * 512.0);
        return (uint8_t)(sign | (uint8_t)m);
    } else {
        int ex;
        double frac = frexp(a, &ex);            /* a = frac * 2^ex, frac in [0.5,1) */
        int e = ex - 1;                         /* a = (2*frac) * 2^e, 2*frac in [1,2) */
        double q = round_half_even((2.0 * frac - 1.0) * 8.0);
        if (q == 8.0) { q = 0.0; e += 1; }
        /* a < 448 keeps (e, q) at or below (8, 6), the largest finite code */
        return (uint8_t)(sign | (uint8_t)(((e + 7) << 3) | (int)q));
    }
}

double mo_bf16_decode(uint16_t bits)
{
    uint32_t u = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* ---------------------------------------------------------------------------------
 * Dynamic group quantisation: the input activations (Sec. 3.3, "Overlapping metadata
 * preparation with input quantization") and the SwiGLU output before the down
 * projection (Sec. 3.3, "Overlapping epilogues": activation, output-scale reduction and
 * cast to the down-projection input) are both quantised per 128-element group.
 * ------------------------------------------------------------------------------- */
void mo_quantize_group(const float* v, int n, uint8_t* q, float* s)
{
    float amax = 0.0f;
    float scale;
    int i;
    for (i = 0; i < n; ++i) {
        float a = fabsf(v[i]);
        if (a > amax) amax = a;
    }
    scale = amax / 448.0f;                       /* IEEE fp32 division */
    if (amax == 0.0f || scale == 0.0f) {
        *s = 0.0f;
        for (i = 0; i < n; ++i) q[i] = 0x00;
        return;
    }
    *s = scale;
    for (i = 0; i < n; ++i) {
        float r = v[i] / scale;                  /* IEEE fp32 division, then RNE to E4M3 */
        q[i] = mo_e4m3_encode(r);
    }
}

/* ---------------------------------------------------------------------------------
 * Router (Sec. 3.3, "Overlapping input fetch with router-logits computation").
 * ------------------------------------------------------------------------------- */
void mo_router_logits(int T, int H, int E, const uint16_t* x_bf16, const uint16_t* rw_bf16,
                      const float* bias, double* logits)
{
    int t, e, h;
    for (t = 0; t < T; ++t) {
        for (e = 0; e < E; ++e) {
            double acc = 0.0;
            for (h = 0; h < H; ++h)
                acc += mo_bf16_decode(x_bf16[(size_t)t * H + h]) *
                       mo_bf16_decode(rw_bf16[(size_t)e * H + h]);
            if (bias) acc += (double)bias[e];
            logits[(size_t)t * E + e] = acc;
        }
    }
}

/* ---------------------------------------------------------------------------------
 * Softmax routing and top-k (Sec. 4.1: the Qwen shapes use softmax routing, eight
 * experts per token).  Selection by repeated arg-max: the largest logit not yet taken,
 * the lowest expert index among equal logits.
 * ------------------------------------------------------------------------------- */
void mo_select(int T, int E, int k, int renorm, const double* logits, int32_t* ids, double* w)
{
    int t, j, e;
    char* taken = (char*)malloc((size_t)E);
    for (t = 0; t < T; ++t) {
        const double* l = logits + (size_t)t * E;
        double m = l[0], denom_all = 0.0, denom_sel = 0.0;
        memset(taken, 0, (size_t)E);
        for (j = 0; j < k; ++j) {
            int best = -1;
            for (e = 0; e < E; ++e) {
                if (taken[e]) continue;
                if (best < 0 || l[e] > l[best]) best = e;
            }
            taken[best] = 1;
            ids[(size_t)t * k + j] = best;
        }
        for (e = 1; e < E; ++e) if (l[e] > m) m = l[e];
        for (e = 0; e < E; ++e) denom_all += exp(l[e] - m);
        for (j = 0; j < k; ++j) denom_sel += exp(l[ids[(size_t)t * k + j]] - m) / denom_all;
        for (j = 0; j < k; ++j) {
            double p = exp(l[ids[(size_t)t * k + j]] - m) / denom_all;
            w[(size_t)t * k + j] = renorm ? p / denom_sel : p;
        }
    }
    free(taken);
}

/* ---------------------------------------------------------------------------------
 * Sigmoid routing with an expert-selection bias (Sec. 4.1: DeepSeek-V3.1 and GLM-5.2,
 * routed scaling factor 2.5).  Each expert's affinity is the logistic function of its
 * logit; the per-expert bias is added for ranking only; the selected affinities are
 * normalised over the selection and scaled.
 * ------------------------------------------------------------------------------- */
void mo_select_sigmoid(int T, int E, int k, const double* logits, const float* sel_bias, double scale,
                       int32_t* ids, double* w)
{
    int t, j, e;
    char* taken = (char*)malloc((size_t)E);
    double* a = (double*)malloc(sizeof(double) * (size_t)E);
    double* score = (double*)malloc(sizeof(double) * (size_t)E);
    for (t = 0; t < T; ++t) {
        double sum = 0.0;
        for (e = 0; e < E; ++e) {
            a[e] = 1.0 / (1.0 + exp(-logits[(size_t)t * E + e]));
            score[e] = a[e] + (sel_bias ? (double)sel_bias[e] : 0.0);
        }
        memset(taken, 0, (size_t)E);
        for (j = 0; j < k; ++j) {
            int best = -1;
            for (e = 0; e < E; ++e) {
                if (taken[e]) continue;
                if (best < 0 || score[e] > score[best]) best = e;
            }
            taken[best] = 1;
            ids[(size_t)t * k + j] = best;
            sum += a[best];
        }
        for (j = 0; j < k; ++j) w[(size_t)t * k + j] = scale * a[ids[(size_t)t * k + j]] / sum;
    }
    free(taken);
    free(a);
    free(score);
}

/* ---------------------------------------------------------------------------------
 * The operator.
 * ------------------------------------------------------------------------------- */
static double silu(double g) { return g / (1.0 + exp(-g)); }

int mo_forward(int T, int H, int E, int I, int k, int renorm,
               const uint16_t* x_bf16, const uint16_t* rw_bf16, const float* bias,
               const uint8_t* const* w13, const float* const* w13s,
               const uint8_t* const* w2, const float* const* w2s,
               const int32_t* ids_in, const double* w_in,
               double* ref, mo_debug_t* dbg)
{
    return mo_forward_policy(T, H, E, I, k, renorm, MO_ROUTING_SOFTMAX, NULL, 1.0, x_bf16, rw_bf16, bias,
                             w13, w13s, w2, w2s, ids_in, w_in, ref, dbg);
}

int mo_forward_policy(int T, int H, int E, int I, int k, int renorm, int policy, const float* sel_bias,
                      double scale, const uint16_t* x_bf16, const uint16_t* rw_bf16, const float* bias,
                      const uint8_t* const* w13, const float* const* w13s,
                      const uint8_t* const* w2, const float* const* w2s,
                      const int32_t* ids_in, const double* w_in,
                      double* ref, mo_debug_t* dbg)
{
    const int HB = H / 128, IB = I / 128;
    int t, j, g, n, kb, kk, i, hh;
    int32_t* ids;
    double* wts;
    uint8_t* xq;
    float* xs;
    double *h, *act, *y;
    uint8_t* aq;
    float* as;
    float* tmp;
    double dec[256];

    if (T < 0 || H <= 0 || I <= 0 || E <= 0 || H % 128 || I % 128) return -1;
    if (k < 1 || k > E) return -1;
    if ((ids_in == NULL) != (w_in == NULL)) return -1;
    if (policy == MO_ROUTING_SOFTMAX) {
        if (sel_bias || scale != 1.0) return -1;
    } else if (policy == MO_ROUTING_SIGMOID_BIAS) {
        if (!(scale > 0.0)) return -1;
    } else {
        return -1;
    }
    if (T == 0) return 0;

    for (n = 0; n < 256; ++n) dec[n] = mo_e4m3_decode((uint8_t)n);

    ids = (int32_t*)malloc(sizeof(int32_t) * (size_t)T * k);
    wts = (double*)malloc(sizeof(double) * (size_t)T * k);
    xq = (uint8_t*)malloc((size_t)T * H);
    xs = (float*)malloc(sizeof(float) * (size_t)T * HB);
    h = (double*)malloc(sizeof(double) * 2 * (size_t)I);
    act = (double*)malloc(sizeof(double) * (size_t)I);
    aq = (uint8_t*)malloc((size_t)I);
    as = (float*)malloc(sizeof(float) * (size_t)IB);
    y = (double*)malloc(sizeof(double) * (size_t)H);
    tmp = (float*)malloc(sizeof(float) * 128);

    /* 1. routing: logits, softmax or sigmoid selection, top-k (or the injected selection) */
    if (ids_in) {
        memcpy(ids, ids_in, sizeof(int32_t) * (size_t)T * k);
        memcpy(wts, w_in, sizeof(double) * (size_t)T * k);
    } else {
        double* logits = (double*)malloc(sizeof(double) * (size_t)T * E);
        mo_router_logits(T, H, E, x_bf16, rw_bf16, bias, logits);
        if (policy == MO_ROUTING_SOFTMAX) mo_select(T, E, k, renorm, logits, ids, wts);
        else mo_select_sigmoid(T, E, k, logits, sel_bias, scale, ids, wts);
        free(logits);
    }
    for (t = 0; t < T * k; ++t) {
        int e = ids[t];
        if (e < 0 || e >= E || !w13[e] || !w13s[e] || !w2[e] || !w2s[e]) {
            free(ids); free(wts); free(xq); free(xs); free(h); free(act); free(aq); free(as); free(y); free(tmp);
            return -1;
        }
    }

    /* 2. per-token, per-128-group input quantisation */
    for (t = 0; t < T; ++t) {
        for (g = 0; g < HB; ++g) {
            for (i = 0; i < 128; ++i)
                tmp[i] = (float)mo_bf16_decode(x_bf16[(size_t)t * H + g * 128 + i]);
            mo_quantize_group(tmp, 128, xq + (size_t)t * H + g * 128, xs + (size_t)t * HB + g);
        }
    }

    for (t = 0; t < T; ++t)
        for (hh = 0; hh < H; ++hh) ref[(size_t)t * H + hh] = 0.0;

    /* 3. every (token, selected expert) pair, token-major */
    for (t = 0; t < T; ++t) {
        for (j = 0; j < k; ++j) {
            const int e = ids[(size_t)t * k + j];
            const size_t p = (size_t)t * k + j;
            const uint8_t* W13 = w13[e];
            const float* S13 = w13s[e];
            const uint8_t* W2 = w2[e];
            const float* S2 = w2s[e];

            /* gate/up projection, Eq. 9 in its standard orientation: for each output row n
             * the 128-deep block products are scaled by the weight block scale and the
             * token's group scale, then summed over blocks */
            for (n = 0; n < 2 * I; ++n) {
                double acc = 0.0;
                for (kb = 0; kb < HB; ++kb) {
                    double blk = 0.0;
                    for (kk = 0; kk < 128; ++kk) {
                        const int col = kb * 128 + kk;
                        blk += dec[W13[(size_t)n * H + col]] * dec[xq[(size_t)t * H + col]];
                    }
                    acc += blk * (double)S13[(size_t)(n / 128) * HB + kb] * (double)xs[(size_t)t * HB + kb];
                }
                h[n] = acc;
            }
            /* SwiGLU: rows [0,I) are the gate, rows [I,2I) the up projection */
            for (i = 0; i < I; ++i) act[i] = silu(h[i]) * h[I + i];
            /* requantisation of fp32(act) per 128-group */
            for (g = 0; g < IB; ++g) {
                for (i = 0; i < 128; ++i) tmp[i] = (float)act[g * 128 + i];
                mo_quantize_group(tmp, 128, aq + g * 128, as + g);
            }
            /* down projection */
            for (hh = 0; hh < H; ++hh) {
                double acc = 0.0;
                for (kb = 0; kb < IB; ++kb) {
                    double blk = 0.0;
                    for (kk = 0; kk < 128; ++kk) {
                        const int col = kb * 128 + kk;
                        blk += dec[W2[(size_t)hh * I + col]] * dec[aq[col]];
                    }
                    acc += blk * (double)S2[(size_t)(hh / 128) * IB + kb] * (double)as[kb];
                }
                y[hh] = acc;
            }
            /* top-k weighted reduction */
            for (hh = 0; hh < H; ++hh) ref[(size_t)t * H + hh] += wts[p] * y[hh];

            if (dbg) {
                if (dbg->h) memcpy(dbg->h + p * 2 * I, h, sizeof(double) * 2 * (size_t)I);
                if (dbg->act) memcpy(dbg->act + p * I, act, sizeof(double) * (size_t)I);
                if (dbg->aq) memcpy(dbg->aq + p * I, aq, (size_t)I);
                if (dbg->as) memcpy(dbg->as + p * IB, as, sizeof(float) * (size_t)IB);
                if (dbg->y) memcpy(dbg->y + p * H, y, sizeof(double) * (size_t)H);
            }
        }
    }

    if (dbg) {
        if (dbg->ids) memcpy(dbg->ids, ids, sizeof(int32_t) * (size_t)T * k);
        if (dbg->w) memcpy(dbg->w, wts, sizeof(double) * (size_t)T * k);
        if (dbg->xq) memcpy(dbg->xq, xq, (size_t)T * H);
        if (dbg->xs) memcpy(dbg->xs, xs, sizeof(float) * (size_t)T * HB);
    }
    free(ids); free(wts); free(xq); free(xs); free(h); free(act); free(aq); free(as); free(y); free(tmp);
    return 0;
}
