// Internal interface between the host runtime (monomoe_api.hip) and the persistent
// kernels (monomoe_kernel.hip, monomoe_kernel_mt.hip).  Not installed; not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace monomoe {

constexpr int kComputeWaves = 4;              // wavefronts that stream weights and run MFMAs
constexpr int kWaves = kComputeWaves + 1;     // + one helper wavefront (epilogues, flags)
constexpr int kThreads = kWaves * 64;
constexpr int kTMax = 16;                     // tokens per pass: one 16-wide MFMA N tile
constexpr int kTLimit = 64;                   // tokens per forward (larger T runs in passes)
constexpr int kKMax = 16;                     // top-k bound
constexpr int kEMax = 512;                    // experts bound (8 logits per lane in top-k)
constexpr int kUMax = kTMax * kKMax;          // active experts bound (T*k, also <= E)
constexpr int kSlotsMin = 4;                  // partial-sum hand-off slots per workgroup:
constexpr int kSlotsMax = 32;                 //   a power of two in [min, max], as LDS allows

constexpr int kGridMax = 1024;                // persistent workgroups at most
constexpr int kUpBlockLogMax = 3;             // gate/up units per deal at most: 2^3 (schedule)

// Multi-tile kernel (more tokens than one 16-wide N tile): tokens are compacted per
// active expert and processed in segments of at most R tokens, each segment on up to
// kNtMax N tiles.
constexpr int kPMax = kTLimit * kKMax;        // token-expert pairs per forward
constexpr int kNtMax = kTLimit / 16;          // N tiles per segment
constexpr int kQMax = 640;                    // segments per forward

// Control words at the head of the workspace (uint32 each).
//  * status: sticky device status (kDev*).
//  * epoch[wg]: launches this workgroup has completed.  All workgroups advance in
//    lockstep, so a launch's tag (epoch + 1) is the same everywhere; cross-workgroup
//    data (logits, SiLU activations, output contributions) is written as 8-byte words
//    {value, tag}, and a reader knows a word is from this launch when its tag matches.
//    Nothing is reset between launches.
//  * ids: the multi-tile kernel's exchange of selected experts, {expert id, tag} words
//    [T*k] (8-byte aligned).
enum : int {
    kCtlStatus = 0,
    kCtlEpoch = 64,                       // [kGridMax]
    kCtlIds = kCtlEpoch + kGridMax,       // [2 * kPMax]
};
static_assert(kCtlIds % 2 == 0, "8-byte words");
constexpr int ctl_words() { return kCtlIds + 2 * kPMax; }

enum : uint32_t { kDevOk = 0, kDevTimeout = 1, kDevBadIds = 2, kDevOverflow = 3 };

// Routing policies (the same values as MONOMOE_ROUTING_* of the C ABI).
enum : int32_t { kRouteSoftmax = 0, kRouteSigmoidBias = 1 };

// Phase stamps (test hook): per workgroup, s_memrealtime at these points.
constexpr int kStamps = 24;
enum : int {
    kStEntry = 0, kStIssued, kStFirstData, kStMeta, kStUpComputed, kStUpDone, kStFirstAq, kStDownDone,
    kStExit, kStFirstMfma, kStComputeDone, kStRouter, kStQuant, kStTopk, kStReduced, kStLogits, kStSelected,
    kStSeek, kStLbase, kStMask,
};

struct KParams {
    // operator inputs/outputs (caller-owned)
    const uint16_t* x;        // bf16 [T,H]
    const uint16_t* rw;       // bf16 [E,H]
    const float* bias;        // fp32 [E] logit bias or null
    const float* sel_bias;    // fp32 [E] expert-selection bias (sigmoid routing) or null
    const uint8_t* w13;       // e4m3 [E,2I,H]
    const float* w13s;        // fp32 [E,2I/128,H/128]
    const uint8_t* w2;        // e4m3 [E,H,I]
    const float* w2s;         // fp32 [E,H/128,I/128]
    uint16_t* out;            // bf16 [T,H]
    // plan workspace
    uint32_t* ctl;            // control words
    uint64_t* logits;         // [T,E]   {fp32 logit, tag}
    uint64_t* xqw;            // [T,H/4] {four E4M3 input codes, tag}
    uint64_t* xsw;            // [T,H/128] {fp32 input scale, tag}
    uint64_t* act;            // [T*k,I] {fp32 SiLU(gate)*up, tag}
    uint64_t* contrib;        // [T*k,S,H] {fp32 routing-weighted expert output, tag}; S = 1,
                              //   or the down projection's K slices (multi-tile kernel)
    // test hooks (null when unused)
    int32_t* d_ids;
    float* d_w;
    uint8_t* d_xq;
    float* d_xs;
    float* d_act;
    uint8_t* d_aq;
    float* d_as;
    float* d_out;
    const int32_t* inj_ids;
    const float* inj_w;
    uint64_t* stamps;         // [grid][kStamps]
    uint64_t spin_limit;      // 100 MHz ticks
    int16_t fail_flag;
    uint16_t jitter;          // race-perturbation seed (0: off)
    // runtime shape and LDS layout
    int32_t T, E, k, renorm;
    int32_t policy;           // MONOMOE_ROUTING_SOFTMAX / MONOMOE_ROUTING_SIGMOID_BIAS
    float route_scale;        // routed scaling factor (sigmoid routing)
    int16_t naq;              // requantised-act LDS buffers (2 = double buffered, 1)
    int16_t nslots;           // partial-sum hand-off slots (power of two)
    // single-tile kernel's work partition (schedule; monomoe_partition.h)
    uint8_t up_lb;            // gate/up units per deal: 2^up_lb
    uint8_t pad0;
    uint16_t dn_grid;         // workgroups with down units (the first dn_grid of the grid)
    // multi-tile kernel only (packed into the struct's tail padding)
    uint8_t mt_rows;          // R: tokens per segment at most (<= kTLimit)
    uint8_t mt_tiles;         // N tiles per hand-off slot entry: ceil(R / 16)
    uint16_t mt_pool;         // quantised-input LDS rows (>= R), used as a ring over segments
};
static_assert(sizeof(KParams) == 256, "kernel argument block");

// One compiled (H, I) specialisation, in every weight-ring depth of kRings.
constexpr int kRings[2] = {2, 4};
struct KernelVariant {
    int ring;
    const void* fn;                                          // __global__ symbol
    void (*launch)(const KParams&, int grid, size_t lds, hipStream_t);
    // the same kernel specialised for one token (T = 1; null: none), with the same LDS layout
    const void* fn1;
    void (*launch1)(const KParams&, int grid, size_t lds, hipStream_t);
};
struct KernelEntry {
    int H, I;
    int ring_default;                                        // the shape's default depth
    KernelVariant v[2];                                      // one per kRings entry
};

const KernelEntry* find_kernel(int H, int I);
const KernelVariant* find_mt_kernel(int H, int I);           // the multi-tile kernel of a shape
int kernel_count();
const KernelEntry* kernel_at(int i);

// Dynamic LDS: the phase-aliased region (quantised input during gate/up; `naq`
// requantised-act buffers during down) followed by the partial-sum hand-off slots.
// Code rows are padded by 16 bytes; the scale arrays always have kTMax rows (rows of
// absent or unrouted tokens hold 0, which zeroes their MFMA columns); every buffer
// starts 16-byte aligned.
__host__ __device__ inline int lds_up_bytes(int H, int T) { return T * (H + 16) + kTMax * (H / 128) * 4; }
__host__ __device__ inline int lds_aq_buffer_bytes(int I, int T) {
    return (T * (I + 16) + kTMax * (I / 128) * 4 + 15) & ~15;
}
__host__ __device__ inline int lds_region_bytes(int H, int I, int T, int naq) {
    const int up = lds_up_bytes(H, T);
    const int dn = naq * lds_aq_buffer_bytes(I, T);
    const int m = up > dn ? up : dn;
    return (m + 15) & ~15;
}
// per slot, one 16x16 fp32 partial tile per compute wavefront
__host__ __device__ inline int lds_partials_bytes(int nslots) { return nslots * kComputeWaves * 64 * 16; }
__host__ __device__ inline int lds_dynamic_bytes(int H, int I, int T, int naq, int nslots) {
    return lds_region_bytes(H, I, T, naq) + lds_partials_bytes(nslots);
}

// Multi-tile kernel LDS.  The down projection runs over K slices of DKB 128-deep blocks:
// the largest even divisor of I/128 not above 16 (a slice of every segment's tokens is
// what the requantised-act buffer holds).  Region: during gate/up a ring of `pool`
// quantised-input rows plus their scale rows (and one zero scale row for absent token
// columns); during down two requantised-act buffers of R rows of one slice (plus a zero
// scale row).  Then the partial-sum slots, `tiles` 16x16 fp32 tiles per compute wavefront.
__host__ __device__ constexpr int mt_slice_blocks(int IB) {
    int d = IB < 16 ? IB : 16;
    while (d > 2 && (IB % d != 0 || d % 2 != 0)) --d;
    return d;
}
__host__ __device__ inline int mt_up_bytes(int H, int pool) { return pool * (H + 16) + (pool + 1) * (H / 128) * 4; }
__host__ __device__ inline int mt_dn_buffer_bytes(int I, int R) {
    const int dkb = mt_slice_blocks(I / 128);
    return (R * (dkb * 128 + 16) + (R + 1) * dkb * 4 + 15) & ~15;
}
__host__ __device__ inline int mt_region_bytes(int H, int I, int pool, int R) {
    const int up = mt_up_bytes(H, pool), dn = 2 * mt_dn_buffer_bytes(I, R);
    return ((up > dn ? up : dn) + 15) & ~15;
}
__host__ __device__ inline int mt_partials_bytes(int nslots, int tiles) { return nslots * kComputeWaves * tiles * 64 * 16; }

}  // namespace monomoe
