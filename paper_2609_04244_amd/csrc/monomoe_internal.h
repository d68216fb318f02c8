// Internal interface between the host runtime (monomoe_api.hip) and the persistent
// kernel (monomoe_kernel.hip).  Not installed; not part of the C ABI.
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

// Control words at the head of the workspace (uint32 each).
//  * status: sticky device status (kDev*).
//  * epoch[wg]: launches this workgroup has completed.  All workgroups advance in
//    lockstep, so a launch's tag (epoch + 1) is the same everywhere; cross-workgroup
//    data (logits, SiLU activations, output contributions) is written as 8-byte words
//    {value, tag}, and a reader knows a word is from this launch when its tag matches.
//    Nothing is reset between launches.
enum : int {
    kCtlStatus = 0,
    kCtlEpoch = 64,                       // [kGridMax]
};
constexpr int ctl_words() { return kCtlEpoch + kGridMax; }

enum : uint32_t { kDevOk = 0, kDevTimeout = 1, kDevBadIds = 2 };

// Routing policies (the same values as MONOMOE_ROUTING_* of the C ABI).
enum : int32_t { kRouteSoftmax = 0, kRouteSigmoidBias = 1 };

// Phase stamps (test hook): per workgroup, s_memrealtime at these points.
constexpr int kStamps = 24;
enum : int {
    kStEntry = 0, kStIssued, kStFirstData, kStMeta, kStUpComputed, kStUpDone, kStFirstAq, kStDownDone,
    kStExit, kStFirstMfma, kStComputeDone, kStRouter, kStQuant, kStTopk, kStReduced, kStLogits, kStSelected, kStSeek, kStLbase,
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
    uint64_t* contrib;        // [T*k,H] {fp32 routing-weighted expert output, tag}
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
    int32_t fail_flag;
    // runtime shape and LDS layout
    int32_t T, E, k, renorm;
    int32_t policy;           // MONOMOE_ROUTING_SOFTMAX / MONOMOE_ROUTING_SIGMOID_BIAS
    float route_scale;        // routed scaling factor (sigmoid routing)
    int32_t naq;              // requantised-act LDS buffers (2 = double buffered, 1)
    int32_t nslots;           // partial-sum hand-off slots (power of two)
};

// One compiled (H, I) specialisation, in every weight-ring depth of kRings.
constexpr int kRings[2] = {2, 4};
struct KernelVariant {
    int ring;
    const void* fn;                                          // __global__ symbol
    void (*launch)(const KParams&, int grid, size_t lds, hipStream_t);
};
struct KernelEntry {
    int H, I;
    int ring_default;                                        // the shape's default depth
    KernelVariant v[2];                                      // one per kRings entry
};

const KernelEntry* find_kernel(int H, int I);
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

}  // namespace monomoe
