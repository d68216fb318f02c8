/*
 * monomoe.h -- C ABI of the MI355X (gfx950) fused routed-MoE decode operator.
 *
 * The operator is the complete routed Mixture-of-Experts layer of MonoMoE
 * (arXiv 2609.04244) for block-wise FP8 experts, at decode token counts:
 *   router logits -> softmax + top-k -> per-token, per-128-group dynamic E4M3
 *   quantisation of the input -> block-FP8 gate/up projection -> SiLU(gate)*up ->
 *   requantisation -> block-FP8 down projection -> top-k weighted reduction,
 * all inside ONE persistent kernel launch (paper Sec. 3, "MonoMoE Design": a single
 * kernel with four logical stages linked by readiness flags).
 *
 * The operator interface follows the paper's generic form (Sec. 3.4): the model shape
 * is fixed per plan together with a token bound T (the paper's B_max); the token count of
 * a call is a runtime argument up to that bound (monomoe_forward_tokens; monomoe_forward
 * runs exactly T).  Top-k and the renormalisation flag are fixed per plan (the paper makes
 * k a runtime argument: a deviation, since k sizes the routing tables and the workspace);
 * the routing policy and its inputs (softmax or sigmoid routing, optional per-expert
 * logit bias, selection bias, scaling factor) are set on a plan between calls.  X is the
 * input tile, R the routing inputs (router weight and biases), W_gu/W_down the expert
 * weights and S their block scales.
 *
 * Conventions for every entry point:
 *  - All tensor pointers are DEVICE pointers owned by the caller.  The library never
 *    frees them and never keeps them beyond the work it enqueues.
 *  - Tensor pointers must be 16-byte aligned and tensors densely packed, row-major.
 *  - Entry points return MONOMOE_OK (0) or a negative monomoe_status_t.  An argument
 *    error enqueues nothing.
 *  - monomoe_forward(), monomoe_forward_tokens() and monomoe_forward_debug() never
 *    synchronise, never allocate, and enqueue one kernel on the given stream (consecutive
 *    kernels only for a schedule that forces the single-tile kernel on more tokens than
 *    its tile, see monomoe_plan_set_schedule), so they can be captured into a HIP graph
 *    and replayed (the kernel's arguments are fixed at capture; the inputs are read from
 *    the captured pointers at every replay).  A plan owns device workspace: one plan must
 *    not be used by two launches that can overlap (use one plan per stream).
 *  - The kernel reports failures it detects on the device (a bounded wait that expired)
 *    through a status word read with monomoe_plan_status().
 */
#ifndef MONOMOE_H
#define MONOMOE_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* T: tokens per decode step (0..64; T == 0 makes forward a no-op).  Up to one MFMA N
 * tile of tokens (16, or as many as the LDS staging of the shape holds: 9 for the
 * 4096x14336 layer) the single-tile kernel runs; beyond that the multi-tile kernel, which
 * compacts each active expert's tokens into segments of up to R tokens (R from the LDS
 * budget, see monomoe_plan_info) on several N tiles, so the weights of an expert are read
 * once per forward unless more than R tokens select it.  Either way one launch.
 * H: hidden size, I: expert intermediate size, both multiples of 128 from the set of
 * compiled shapes (monomoe_supported_shape()).  E: routed experts (1..512). */
typedef struct {
    int32_t T, H, E, I;
} monomoe_shape_t;

typedef struct monomoe_plan_s* monomoe_plan_t;

typedef enum {
    MONOMOE_OK = 0,
    MONOMOE_ERR_INVALID = -1,      /* bad argument: null/misaligned pointer, bad shape, bad topk */
    MONOMOE_ERR_UNSUPPORTED = -2,  /* valid but not compiled: (H,I) pair, T > 64, E > 512     */
    MONOMOE_ERR_OCCUPANCY = -3,    /* the persistent grid cannot be fully resident             */
    MONOMOE_ERR_HIP = -4,          /* a HIP runtime call failed                                */
    MONOMOE_ERR_TIMEOUT = -5       /* device: a bounded readiness wait expired                 */
} monomoe_status_t;

/* Create a plan for one shape.  topk in [1, E] and topk <= 16; renorm != 0 renormalises
 * the selected softmax probabilities to sum to 1.  Allocates and zeroes the plan's device
 * workspace on the current device (synchronously) and picks the persistent grid:
 * one workgroup per compute unit, after checking that the occupancy calculator allows
 * at least one per CU for the plan's LDS footprint (readiness waits need every
 * workgroup resident; paper Sec. 3.2 "Persistent residency").  *plan_out is set only
 * on success. */
int monomoe_plan(const monomoe_shape_t* shape, int topk, int renorm, monomoe_plan_t* plan_out);

/* Release a plan and its workspace.  The caller makes sure no enqueued launch that uses
 * the plan is still pending.  NULL is ignored. */
void monomoe_plan_destroy(monomoe_plan_t plan);

/* Optional routing input (paper Sec. 3.4: R, the operator's routing inputs, beside the
 * router weight): a per-expert fp32 bias [E] (device pointer, or NULL to remove) added to
 * the router logits before softmax and selection, so it changes both the selected experts
 * and their weights.  The pointer is read by every later forward.  Returns
 * MONOMOE_ERR_INVALID for a NULL plan or a pointer that is not 16-byte aligned. */
int monomoe_plan_set_router_bias(monomoe_plan_t plan, const float* bias);

/* Routing policy (paper Sec. 4.1: softmax routing for the Qwen models; sigmoid routing
 * with an expert-selection bias and a routed scaling factor of 2.5 for DeepSeek-V3.1 and
 * GLM-5.2; Sec. 3.4 lists the policy p among the operator's runtime parameters).
 *   MONOMOE_ROUTING_SOFTMAX (the default): top-k of the logits, softmax weights,
 *     renormalised over the selection when the plan's renorm flag is set.  sel_bias must
 *     be NULL and scale 1.
 *   MONOMOE_ROUTING_SIGMOID_BIAS: affinity a_e = 1/(1+exp(-logit_e)); experts ranked by
 *     a_e + sel_bias[e] (fp32 [E] device pointer, or NULL for none; lower index on ties);
 *     w_j = scale * a_{e_j} / sum of the selected affinities (the renorm flag is ignored).
 *     scale must be finite and > 0.
 * A logit bias set with monomoe_plan_set_router_bias applies under either policy.  The
 * sel_bias pointer is read by every later forward.  Returns MONOMOE_ERR_INVALID (plan
 * unchanged) on a bad policy, scale, pointer alignment or a softmax bias/scale. */
enum { MONOMOE_ROUTING_SOFTMAX = 0, MONOMOE_ROUTING_SIGMOID_BIAS = 1 };
int monomoe_plan_set_routing(monomoe_plan_t plan, int policy, const float* sel_bias, float scale);

/* The operator (paper Sec. 3.4 interface, Eq. 9 weight-major projections):
 *   x         bf16  [T,H]                 input token tile
 *   router_w  bf16  [E,H]                 logits = x . router_w^T (+ bias)
 *   w13       e4m3fn bytes [E,2I,H]       rows [0,I) gate, rows [I,2I) up, K (=H) contiguous
 *   w13_scale fp32  [E,2I/128,H/128]      dequantised weight = decode(byte) * block scale
 *   w2        e4m3fn bytes [E,H,I]        K (=I) contiguous
 *   w2_scale  fp32  [E,H/128,I/128]
 *   out       bf16  [T,H]                 fully overwritten (round-to-nearest-even)
 * Enqueues one kernel on `stream`. */
int monomoe_forward(monomoe_plan_t plan, const void* x, const void* router_w,
                    const void* w13, const float* w13_scale,
                    const void* w2, const float* w2_scale,
                    void* out, hipStream_t stream);

/* The operator on T tokens, for any T in [0, the plan's T], without re-planning (paper
 * Sec. 3.4: the decode batch size B <= B_max is a runtime argument of the operator; here the
 * plan's T is B_max).  x is bf16 [T,H] and out bf16 [T,H]; every other argument and the
 * asynchrony are as for monomoe_forward, and T == 0 enqueues nothing.  The kernel is chosen per
 * call: when the plan's T needs the multi-tile kernel, a call with at most one single-tile
 * kernel tile of tokens takes the single-tile kernel instead (unless the plan's schedule
 * forces a kernel, or the layer's down projection is sliced, see monomoe_plan_info).  The
 * plan's workspace, sized for its T, serves every smaller T.  Returns MONOMOE_ERR_INVALID
 * (nothing enqueued) for T outside [0, the plan's T]. */
int monomoe_forward_tokens(monomoe_plan_t plan, int32_t T, const void* x, const void* router_w,
                           const void* w13, const float* w13_scale,
                           const void* w2, const float* w2_scale,
                           void* out, hipStream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): the operator of monomoe_forward without a
 * plan, allocating nothing.  Its workspace is one file-scope device array of the library
 * (32 MiB per GPU it runs on, held until the process ends; set up on the first call on each
 * device); the caller passes inputs and outputs only:
 *   shape, topk, renorm  as for monomoe_plan; softmax routing;
 *   bias                 fp32 [E] logit bias (device, 16-byte aligned) or NULL, as for
 *                        monomoe_plan_set_router_bias;
 *   x .. out, stream     as for monomoe_forward;
 *   status               int32 device word or NULL: receives, in stream order after the
 *                        operator, MONOMOE_OK or the device-side failure of this call
 *                        (MONOMOE_ERR_TIMEOUT, MONOMOE_ERR_INVALID for a bad expert id).
 * Enqueues the operator's kernel(s) and one single-workgroup status kernel; never
 * synchronises and calls no allocating routine.  Every call on one GPU shares that GPU's
 * array, which keeps the last call's contents (the tagged exchange needs no clearing; the
 * status word is cleared by the status kernel): calls that can overlap on one GPU (other
 * streams, other host threads) race and must be serialised by the caller.  Returns
 * MONOMOE_ERR_UNSUPPORTED when the shape's workspace exceeds 32 MiB (e.g. 64 tokens of the
 * 4096x14336 layer), and the argument errors of monomoe_plan and monomoe_forward. */
int monomoe_forward_noalloc(const monomoe_shape_t* shape, int topk, int renorm, const float* bias,
                            const void* x, const void* router_w,
                            const void* w13, const float* w13_scale,
                            const void* w2, const float* w2_scale,
                            void* out, int32_t* status, hipStream_t stream);

/* Test hooks.  Every pointer may be NULL.  Pair index p = t*topk + j.
 *   topk_ids  int32 [T,topk]      selected experts, in selection order (written)
 *   topk_w    fp32  [T,topk]      their routing weights (written)
 *   xq        u8    [T,H]         E4M3 codes of the quantised input (written)
 *   xs        fp32  [T,H/128]     input group scales (written)
 *   act       fp32  [T*topk,I]    SiLU(gate)*up before requantisation (written)
 *   aq        u8    [T*topk,I]    requantised activation codes (written)
 *   as        fp32  [T*topk,I/128] requantisation scales (written)
 *   out_f32   fp32  [T,H]         the weighted sum before rounding to bf16 (written)
 *   topk_ids_in / topk_w_in       [T,topk] replace the kernel's own selection (read);
 *                                 both or neither; ids distinct per token, in [0,E)
 *   stamps    u64   [grid,24]     per-workgroup s_memrealtime (100 MHz) stamps at phase
 *                                 boundaries, for latency breakdowns (written; with
 *                                 several single-tile passes, those of the last pass)
 *   spin_limit_ticks              bound of every readiness wait in 100 MHz ticks
 *                                 (0 = the default of 2 s)
 *   fail_flag                     nonzero makes every workgroup wait on a condition that
 *                                 never holds (bounded by the spin limit), so the kernel
 *                                 takes its timeout path and reports MONOMOE_ERR_TIMEOUT
 *                                 through monomoe_plan_status().
 *   jitter_seed                   race perturbation: nonzero (at most 65535) inserts
 *                                 pseudo-random pauses of 0 to 2.55 us, a function of the
 *                                 seed, at every cross-wavefront and cross-workgroup
 *                                 hand-off point (partial sums, activation and contribution
 *                                 stores, activation polls, output reduction, kernel
 *                                 entry), so the readiness protocol runs under orders of
 *                                 arrival it rarely sees; results must not change.  0: off.
 *                                 MONOMOE_ERR_INVALID above 65535. */
typedef struct {
    int32_t* topk_ids;
    float* topk_w;
    uint8_t* xq;
    float* xs;
    float* act;
    uint8_t* aq;
    float* as;
    float* out_f32;
    const int32_t* topk_ids_in;
    const float* topk_w_in;
    uint64_t* stamps;
    uint64_t spin_limit_ticks;
    int32_t fail_flag;
    uint32_t jitter_seed;
} monomoe_debug_t;

int monomoe_forward_debug(monomoe_plan_t plan, const void* x, const void* router_w,
                          const void* w13, const float* w13_scale,
                          const void* w2, const float* w2_scale,
                          void* out, const monomoe_debug_t* dbg, hipStream_t stream);

/* Measurement hook: monomoe_forward with the kernel launched through hipExtLaunchKernel,
 * so that `start` and `stop` (caller-created hipEvents, both non-NULL) take the dispatch's
 * own begin and end timestamps instead of the stream positions around it; the elapsed
 * time between them is the kernel duration that a kernel trace reports (with several
 * token passes: from the first pass's begin to the last pass's end).  Same arguments,
 * errors and asynchrony as monomoe_forward. */
int monomoe_forward_timed(monomoe_plan_t plan, const void* x, const void* router_w,
                          const void* w13, const float* w13_scale,
                          const void* w2, const float* w2_scale,
                          void* out, hipEvent_t start, hipEvent_t stop, hipStream_t stream);

/* Device-side status of the plan's last launches: MONOMOE_OK or MONOMOE_ERR_TIMEOUT.
 * Blocking: copies the status word to the host after a device synchronisation.  The
 * status is sticky until monomoe_plan_reset(). */
int monomoe_plan_status(monomoe_plan_t plan);

/* Zero the plan's workspace: the sticky status word, the launch epochs and the tagged
 * exchange buffers (needed after a device-side error, which can leave workgroups out of
 * step).  Blocking. */
int monomoe_plan_reset(monomoe_plan_t plan);

/* Launch geometry and footprint of a plan, for tests and benchmarks. */
typedef struct {
    int32_t grid;            /* persistent workgroups                       */
    int32_t block;           /* threads per workgroup                       */
    int32_t lds_bytes;       /* dynamic + static LDS per workgroup          */
    int32_t occupancy;       /* workgroups per CU the occupancy API allows  */
    int32_t num_cus;
    int64_t workspace_bytes;
    int32_t scratch_bytes;   /* per-thread private (scratch) memory of the kernel: 0 when
                                all of its state lives in registers and LDS            */
    int32_t ring;            /* weight-ring depth of the current schedule             */
    int32_t tokens_per_pass; /* tokens one launch processes (T larger runs in passes) */
    int32_t multi_tile;      /* 1 when the multi-tile kernel runs, else 0             */
    int32_t group_tokens;    /* multi-tile: R, the most tokens of one expert segment  */
    int32_t down_slices;     /* multi-tile: K slices of the down projection           */
    int32_t up_block;        /* single-tile: gate/up units per deal of the schedule   */
    int32_t down_grid;       /* single-tile: workgroups with down units               */
} monomoe_plan_info_t;

int monomoe_plan_info(monomoe_plan_t plan, monomoe_plan_info_t* info);

/* Schedule of a plan (paper Sec. 3.4: each shape's kernels are precompiled for a set of
 * schedules and serving uses a fixed, offline-tuned one).  Here a schedule is
 *   grid: persistent workgroups, 1 .. CUs x occupancy (0 = one per CU, the default);
 *   ring: weight-prefetch depth in 256-deep tasks per compute wavefront, 2 or 4 (0 = the
 *         shape's default); the multi-tile kernel has depth 2 only;
 *   kernel: MONOMOE_KERNEL_AUTO (0: single-tile up to its tile, multi-tile beyond),
 *         MONOMOE_KERNEL_SINGLE (token passes of one tile each beyond it) or
 *         MONOMOE_KERNEL_MULTI (also below one tile);
 *   group_tokens: multi-tile only, a cap on R (0 = the largest the LDS holds), e.g. to
 *         study segment splitting;
 *   general_only: single-tile only; 0 (default) runs passes of one token on the kernel's
 *         one-token specialisation (the selected experts are the active ones, so each
 *         workgroup starts streaming as soon as the experts it needs are ranked), 1 runs
 *         them on the general kernel;
 *   up_block: single-tile only; gate/up units (8 gate + 8 up rows of one expert) dealt to a
 *         workgroup at a time, round-robin over the grid: 1 (0 = the default), 2, 4 or 8.
 *         An expert's I/8 units are spread over about I/(8 up_block) workgroups: the
 *         workgroups per expert of the gate/up phase (the paper's G_up);
 *   down_grid: single-tile only; the workgroups that run the down projection (the first
 *         down_grid of the grid take contiguous ranges of its 16-row units; 0 = the whole
 *         grid), so that an expert's H/16 down units are spread over about down_grid / U
 *         workgroups for U active experts (the paper's G_down).  At most grid.
 * The task depth (256 deep per ring slot) and the single ring running through both phases
 * are fixed by the design (a ring slot is 16 registers; the first down tasks are in flight
 * while the last gate/up tasks compute).  Schedules that differ only in grid, ring,
 * general_only, up_block or down_grid compute bit-identical outputs; the kernel choice and
 * R change the order of fp32 summation only.
 * A new grid resets the plan's workspace (blocking; no launch of the plan may be pending).
 * Returns MONOMOE_ERR_INVALID (plan unchanged) for an out-of-range field, and
 * MONOMOE_ERR_UNSUPPORTED when the requested kernel cannot hold the shape's tiles. */
enum { MONOMOE_KERNEL_AUTO = 0, MONOMOE_KERNEL_SINGLE = 1, MONOMOE_KERNEL_MULTI = 2 };
typedef struct {
    int32_t grid;
    int32_t ring;
    int32_t kernel;
    int32_t group_tokens;
    int32_t general_only;
    int32_t up_block;
    int32_t down_grid;
} monomoe_schedule_t;
int monomoe_plan_set_schedule(monomoe_plan_t plan, const monomoe_schedule_t* sched);

/* Layout of a kernel's LDS for a shape, and the residency check, computed on the host
 * without a device (no HIP call, no allocation): what monomoe_plan and
 * monomoe_plan_set_schedule configure, for capacity planning and for tests of the
 * refusals.  `shape` and `topk` as for monomoe_plan (shape->T: tokens per forward);
 * `kernel` MONOMOE_KERNEL_SINGLE or MONOMOE_KERNEL_MULTI; `lds_total` the LDS bytes a
 * workgroup may use on the device and `lds_static` the kernel's own static LDS;
 * `occupancy` the workgroups per CU that the device's occupancy query reports for the
 * resulting layout; `grid` the persistent workgroups (0: one per CU) on `num_cus` CUs.
 * Returns MONOMOE_ERR_INVALID / MONOMOE_ERR_UNSUPPORTED for the arguments monomoe_plan
 * refuses and for bad sizes, MONOMOE_ERR_UNSUPPORTED when no layout fits the LDS, else
 * fills *out and returns MONOMOE_ERR_OCCUPANCY when the grid cannot be resident at once
 * (occupancy < 1, or grid > num_cus * occupancy: the kernel's cross-workgroup waits need
 * every workgroup resident; Sec. 3.2, persistent residency), MONOMOE_OK otherwise. */
typedef struct {
    int32_t tokens_per_pass; /* token tile of one pass (multi-tile: T)             */
    int32_t group_tokens;    /* multi-tile: tokens per segment R; single-tile: 0   */
    int32_t act_buffers;     /* requantised-activation LDS buffers                  */
    int32_t handoff_slots;   /* partial-sum hand-off slots between the wavefronts   */
    int32_t lds_bytes;       /* dynamic LDS per workgroup                           */
} monomoe_layout_t;

int monomoe_layout(const monomoe_shape_t* shape, int topk, int kernel, int lds_total, int lds_static,
                   int occupancy, int grid, int num_cus, monomoe_layout_t* out);

/* Host-side model check of the single-tile kernel's hand-off protocol (Sec. 3.2: readiness-
 * based hand-offs between resident workgroups, no grid barrier), without a device.  For one
 * routing, every wavefront's synchronisation events are replayed in the order the kernel
 * issues them, with the kernel's own work-partition arithmetic: workgroup barriers, router
 * rows, the input exchange, the selection (with one token: each top-k position published as
 * it is ranked, and the compute wavefronts' quantisation counter), the partial-sum hand-off
 * slots, the requantised-activation buffers (blocking and non-blocking preparation; with
 * single-wavefront down units, the wavefronts' own down epilogues and the progress the helper
 * waits for before reusing a buffer), the activation and contribution words, the output
 * reduction.  A scheduler interleaves the
 * wavefronts in a pseudo-random order drawn from `seed` (0: in index order, one event each)
 * with at most `resident` workgroups resident at once, started in index order (a new one when
 * one ends).  The result says whether every wavefront ran to its end (no deadlock) and counts
 * safety violations: a hand-off slot rewritten before the helper consumed it, a slot
 * consumed that does not hold the expected sums, an activation buffer read while it holds
 * another expert or rewritten while it is read, a unit published twice.  A unit that no
 * workgroup owns shows as a deadlock (its consumers wait forever).
 *   shape, topk      as for monomoe_plan; shape->T <= 16 (one pass)
 *   topk_ids         host int32 [T, topk]: the selection to replay, ids in [0, E), distinct
 *                    per token (the order within a token is its top-k order)
 *   one_token        1: the one-token specialisation (T must be 1); 0: the general kernel
 *   grid, ring       persistent workgroups (<= 1024) and weight-ring depth (2 or 4)
 *   up_block, down_grid  the schedule's work partition (monomoe_plan_set_schedule: 0, 1, 2,
 *                    4 or 8 gate/up units per deal; 0 or 1 .. grid workgroups with down units)
 *   handoff_slots, act_buffers   the LDS layout (monomoe_layout: a power of two <= 32; 1 or 2)
 *   mutate           0 for the kernel's protocol; MONOMOE_SCHEDULE_MUTATE_* bits remove a
 *                    wait or move a step, so that a test can show the check catches the
 *                    resulting race
 * Returns MONOMOE_ERR_INVALID for bad arguments, MONOMOE_ERR_UNSUPPORTED beyond one pass,
 * else fills *out and returns MONOMOE_OK (whatever the verdict). */
#define MONOMOE_SCHEDULE_MUTATE_NO_SLOT_WAIT 1u    /* hand off without waiting for a free slot        */
#define MONOMOE_SCHEDULE_MUTATE_NO_ACT_WAIT 2u     /* read an activation buffer without waiting       */
#define MONOMOE_SCHEDULE_MUTATE_PREFETCH_ONE_BUFFER 4u  /* prefetch the next expert with one buffer */
typedef struct {
    int32_t complete;        /* 1: every wavefront of every workgroup ran to its end          */
    int32_t violations;      /* safety violations seen (0 for a sound protocol)               */
    int32_t first_violation; /* kind of the first: 1 slot overwritten, 2 stale slot consumed,
                                3 buffer read holding another expert, 4 buffer overwritten
                                while read, 5 a unit published twice; 0 none                  */
    int32_t active_experts;  /* expert slots of the routing                                   */
    int64_t events;          /* synchronisation events executed                               */
    int32_t blocked_wg;      /* at a deadlock: a blocked wavefront's workgroup, wavefront    */
    int32_t blocked_wave;    /*   (helper = 4) and its event kind; -1 when complete          */
    int32_t blocked_event;
    int32_t reserved;
} monomoe_schedule_report_t;

int monomoe_schedule_check(const monomoe_shape_t* shape, int topk, const int32_t* topk_ids, int one_token,
                           int grid, int ring, int up_block, int down_grid, int handoff_slots, int act_buffers,
                           int resident, uint32_t seed,
                           uint32_t mutate, monomoe_schedule_report_t* out);

/* 1 if (H, I) is one of the compiled shapes, else 0. */
int monomoe_supported_shape(int32_t H, int32_t I);

/* Static string for a status code. */
const char* monomoe_status_string(int status);

/* Measurement references (not part of the operator).  Plain dwordx4 grid-stride kernels
 * enqueued on `stream`:
 *   monomoe_stream_copy: dst[0,bytes) = src[0,bytes); a kernel of exactly known HBM
 *     traffic (bytes read + bytes written), used to calibrate HBM byte counters.
 *   monomoe_stream_read: reads src[0,bytes); the achievable streaming-read bandwidth,
 *     reported next to the nominal peak.  sink16 is a 16-byte device scratch word that
 *     is written only in a practically impossible case (it keeps the loads alive).
 * Pointers are device pointers, 16-byte aligned; bytes a multiple of 16.
 * MONOMOE_ERR_INVALID otherwise, MONOMOE_ERR_HIP if the launch fails. */
int monomoe_stream_copy(void* dst, const void* src, size_t bytes, hipStream_t stream);
int monomoe_stream_read(const void* src, size_t bytes, void* sink16, hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif
