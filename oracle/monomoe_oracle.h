/*
 * monomoe_oracle.h -- plain, slow, fp64 CPU oracle for the routed-MoE decode operator
 * of MonoMoE (arXiv 2609.04244).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg may load or call this library.  The product path (the HIP kernel
 * behind include/monomoe.h) never calls it, shares no code, header, table or constant
 * generator with it, and must fail loudly rather than fall back to it.
 *
 * What is computed (paper Sec. 3 "MonoMoE Design" and Sec. 4.1 "Experimental Setup"):
 * router logits, softmax + top-k selection (or sigmoid + selection bias), per-token
 * per-128-element dynamic E4M3
 * activation quantisation, the block-FP8 gate/up projection with 128x128 fp32 weight
 * block scales, SiLU(gate)*up, requantisation, the block-FP8 down projection and the
 * top-k weighted reduction.  The weight-major schedule of the paper changes when and
 * where this work runs, not what it computes (Sec. 2.1, the definition of the
 * idealised monokernel), so the oracle is the plain token-major definition.
 *
 * Precision: accumulation in fp64.  Two steps are defined in fp32 on purpose because
 * the quantised bytes are part of the operator's contract: the scale s = amax/448 and
 * the division v/s are IEEE fp32 operations (correctly rounded), followed by
 * round-to-nearest-even into E4M3.
 *
 * Parity pins: every function here is pinned by tests outside this directory against
 * library routines, closed forms and invariants; none is "parity unpinned".
 */
#ifndef MONOMOE_ORACLE_H
#define MONOMOE_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* OCP 8-bit floating point, E4M3FN variant (the "E4M3" format of Sec. 4.1):
 * 1 sign bit, 4 exponent bits (bias 7), 3 mantissa bits, no infinities,
 * S.1111.111 is NaN, largest finite magnitude 448. */
double mo_e4m3_decode(uint8_t code);
/* Round-to-nearest-even into E4M3FN, saturating magnitudes >= 448 to +-448, keeping the
 * sign of zero.  NaN input gives 0x7F. */
uint8_t mo_e4m3_encode(float v);

/* bfloat16 -> value (exact). */
double mo_bf16_decode(uint16_t bits);

/* Dynamic quantisation of one group of n values (Sec. 3.3 and Sec. 4.1: activations
 * are quantised inside the operator at 128-element granularity):
 *   amax = max |v_i|;  s = fl32(amax / 448);  q_i = e4m3(fl32(v_i / s)).
 * amax == 0 (or an s that underflows to 0) gives s = 0 and all codes 0x00. */
void mo_quantize_group(const float* v, int n, uint8_t* q, float* s);

/* Router logits (Sec. 3.3: router logits computed from the input tile):
 *   logits[t*E+e] = sum_h x[t,h] * rw[e,h]  (+ bias[e] when bias != NULL), fp64. */
void mo_router_logits(int T, int H, int E, const uint16_t* x_bf16, const uint16_t* rw_bf16,
                      const float* bias, double* logits);

/* Softmax routing with top-k (Sec. 4.1 "Models and workload"): experts are ranked by
 * logit, descending, equal logits ranked by lower expert index; ids[t*k+j] is the j-th
 * selected expert.  p = softmax over all E logits; renorm != 0 gives
 * w_j = p_{id_j} / sum_j' p_{id_j'}, otherwise w_j = p_{id_j}. */
void mo_select(int T, int E, int k, int renorm, const double* logits, int32_t* ids, double* w);

/* Sigmoid routing with an expert-selection bias and a routed scaling factor (Sec. 4.1:
 * the DeepSeek-V3.1 and GLM-5.2 shapes, scaling factor 2.5; the formulas are those of the
 * cited DeepSeek-V3 report): affinity a_e = 1 / (1 + exp(-logit_e)); experts are ranked by
 * a_e + sel_bias[e] (sel_bias may be NULL = 0), descending, equal scores ranked by lower
 * expert index; the bias steers the selection only:
 *   w_j = scale * a_{id_j} / sum_j' a_{id_j'}. */
void mo_select_sigmoid(int T, int E, int k, const double* logits, const float* sel_bias, double scale,
                       int32_t* ids, double* w);

/* Routing policies of mo_forward_policy. */
enum { MO_ROUTING_SOFTMAX = 0, MO_ROUTING_SIGMOID_BIAS = 1 };

/* Optional intermediate outputs of mo_forward; any pointer may be NULL.
 * Pair index p = t*k + j (token t, j-th selected expert). */
typedef struct {
    int32_t* ids;   /* [T,k]                                   */
    double*  w;     /* [T,k]                                   */
    uint8_t* xq;    /* [T,H]     E4M3 codes of the input        */
    float*   xs;    /* [T,H/128] input scales                   */
    double*  h;     /* [T*k,2I]  gate/up projection (fp64)      */
    double*  act;   /* [T*k,I]   SiLU(gate)*up (fp64)           */
    uint8_t* aq;    /* [T*k,I]   requantised activation codes   */
    float*   as;    /* [T*k,I/128] requantisation scales        */
    double*  y;     /* [T*k,H]   down projection before weighting */
} mo_debug_t;

/* The whole operator.  Expert weights are given per expert through pointer tables so
 * that a caller may hand over only the experts the routing selects (NULL elsewhere):
 *   w13[e] : E4M3 codes [2I,H] row-major, rows [0,I) gate, rows [I,2I) up
 *   w13s[e]: fp32 [2I/128, H/128] block scales, dequant = decode(code) * scale
 *   w2[e]  : E4M3 codes [H,I] row-major
 *   w2s[e] : fp32 [H/128, I/128]
 * ids_in/w_in (both NULL or both set, [T,k]) replace the routing selection.
 * ref: fp64 [T,H] output, the weighted sum before any rounding to bf16.
 * Returns 0, or -1 for invalid arguments (shape not a multiple of 128, k out of
 * range, a selected expert whose weights are NULL). */
int mo_forward(int T, int H, int E, int I, int k, int renorm,
               const uint16_t* x_bf16, const uint16_t* rw_bf16, const float* bias,
               const uint8_t* const* w13, const float* const* w13s,
               const uint8_t* const* w2, const float* const* w2s,
               const int32_t* ids_in, const double* w_in,
               double* ref, mo_debug_t* dbg);

/* mo_forward with the routing policy made explicit: MO_ROUTING_SOFTMAX (renorm as in
 * mo_select; sel_bias must be NULL and scale 1) or MO_ROUTING_SIGMOID_BIAS (mo_select_sigmoid
 * with sel_bias and scale; renorm is ignored).  bias, when set, is added to the logits under
 * either policy. */
int mo_forward_policy(int T, int H, int E, int I, int k, int renorm, int policy, const float* sel_bias,
                      double scale, const uint16_t* x_bf16, const uint16_t* rw_bf16, const float* bias,
                      const uint8_t* const* w13, const float* const* w13s,
                      const uint8_t* const* w2, const float* const* w2s,
                      const int32_t* ids_in, const double* w_in,
                      double* ref, mo_debug_t* dbg);

#ifdef __cplusplus
}
#endif
#endif
