// Device-side building blocks shared by the persistent kernels: coherent and LDS
// memory helpers, exact E4M3 arithmetic, the fp16 MFMA block contraction, bounded
// waits, input quantisation (replicated or exchanged), the router GEMV, top-k and the
// routing weights.  Included by the kernel sources only.
#pragma once

#include "monomoe_internal.h"
#include "monomoe_partition.h"

namespace monomoe {


typedef float v4f __attribute__((ext_vector_type(4)));
typedef int v4i __attribute__((ext_vector_type(4)));
typedef _Float16 v8h __attribute__((ext_vector_type(8)));
typedef _Float16 v2h __attribute__((ext_vector_type(2)));


// ------------------------------------------------------------------------------------
// memory helpers
// ------------------------------------------------------------------------------------
// Agent-scope relaxed atomics compile to sc1 accesses: coherent across XCDs.
template <class Tp>
__device__ __forceinline__ Tp ld_co(const Tp* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <class Tp>
__device__ __forceinline__ void st_co(Tp* p, Tp v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t add_co(uint32_t* p, uint32_t v) {
    return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void compiler_fence() { __atomic_signal_fence(__ATOMIC_SEQ_CST); }
// Wait until every vector-memory operation this wavefront issued has completed
// (s_waitcnt vmcnt(0), other counters untouched).
__device__ __forceinline__ void vm_drain() {
    compiler_fence();
    __builtin_amdgcn_s_waitcnt(0x0F70);
    compiler_fence();
}
// 16-byte coherent accesses through a raw buffer resource with the sc1 cache policy.
constexpr int kCachePolicySc1 = 16;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void* base) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, 0x7FFFFFFF, 0x00020000);
}
__device__ __forceinline__ v4i ld_co16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kCachePolicySc1);
}
// Four consecutive tagged words {fp32 value, tag} from one lane (byte offset `off`, 32-byte
// aligned), written as two 16-byte sc1 stores: each store is one request, so neither of its
// two naturally aligned 8-byte words can tear, and a lane's four words fill one 32-byte
// sector (an 8-byte agent-scope store costs a 32-byte memory write on its own).
__device__ __forceinline__ void st_tagged4(__amdgpu_buffer_rsrc_t r, uint32_t off, uint32_t tag, const v4f& v) {
    const v4i lo = {(int)__float_as_uint(v[0]), (int)tag, (int)__float_as_uint(v[1]), (int)tag};
    const v4i hi = {(int)__float_as_uint(v[2]), (int)tag, (int)__float_as_uint(v[3]), (int)tag};
    __builtin_amdgcn_raw_buffer_store_b128(lo, r, off, 0, kCachePolicySc1);
    __builtin_amdgcn_raw_buffer_store_b128(hi, r, off + 16u, 0, kCachePolicySc1);
}

// LDS flags shared by the wavefronts of a workgroup.  They are accessed through
// LDS-address-space pointers with relaxed ordering: a flag update is preceded by
// s_waitcnt lgkmcnt(0) (this wavefront's LDS writes are done) and LDS executes one
// CU's requests in order, so a reader that sees the flag sees the data.  Neither side
// waits on vmcnt, which would drain the weight stream.
#define LDS_AS __attribute__((address_space(3)))
__device__ __forceinline__ void lgkm_drain() {
    compiler_fence();
    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0), vmcnt/expcnt untouched
    compiler_fence();
}
__device__ __forceinline__ int lds_ld(const int* p) {
    return __hip_atomic_load((const LDS_AS int*)p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ void lds_st(int* p, int v) {
    lgkm_drain();
    __hip_atomic_store((LDS_AS int*)p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ void lds_add(int* p, int v) {
    lgkm_drain();
    __hip_atomic_fetch_add((LDS_AS int*)p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

__device__ __forceinline__ uint64_t now() { return __builtin_amdgcn_s_memrealtime(); }

// Test hook: record a phase stamp for this workgroup (one lane writes).
__device__ __forceinline__ void stamp(uint64_t* stamps, int wg, int which) {
    if (stamps) stamps[wg * kStamps + which] = now();
}

// Race perturbation (compiled into the perturbation build of the library only, which defines
// MONOMOE_RACE_PERTURB): a pseudo-random pause of 0 to 2.55 us (s_memrealtime ticks of 10 ns)
// at a hand-off point, taken at about half of the calls; seed 0 returns at once.  The pause
// depends only on (seed, workgroup, wavefront, site, n), all uniform across the wavefront,
// mixed by the lowbias32 integer hash (C. Wellons, "hash prospector"), so a seed replays the
// same perturbation.  In the product build MONOMOE_PERTURB is empty: its kernels carry no
// trace of the hook.
__device__ __forceinline__ void jitter(uint32_t seed, int wg, int wv, int site, int n) {
    if (seed == 0u) return;
    uint32_t h = seed * 0x9E3779B9u ^ (uint32_t)wg * 0x85EBCA6Bu ^ ((uint32_t)wv << 24) ^ ((uint32_t)site << 20) ^
                 (uint32_t)n;
    h ^= h >> 16;
    h *= 0x7FEB352Du;
    h ^= h >> 15;
    h *= 0x846CA68Bu;
    h ^= h >> 16;
    if (h & 1u) return;
    const uint64_t d = (h >> 8) & 255u;
    const uint64_t t0 = now();
    while (now() - t0 < d) __builtin_amdgcn_s_sleep(1);
}
#ifdef MONOMOE_RACE_PERTURB
#define MONOMOE_PERTURB(site, n) jitter(p.jitter, wg, wv, (site), (n))
#else
#define MONOMOE_PERTURB(site, n) ((void)0)
#endif

// Record the first device-side error; later ones keep the first code.
__device__ __forceinline__ void set_status(uint32_t* status, uint32_t code) {
    uint32_t expected = kDevOk;
    __hip_atomic_compare_exchange_strong(status, &expected, code, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                         __HIP_MEMORY_SCOPE_AGENT);
}

// ------------------------------------------------------------------------------------
// arithmetic helpers
// ------------------------------------------------------------------------------------
__device__ __forceinline__ float bf16_to_f32(uint32_t b) { return __uint_as_float(b << 16); }
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);   // round to nearest even (finite inputs)
    return (uint16_t)(u >> 16);
}

template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), CTRL, 0xF, 0xF, false));
}
template <int CTRL>
__device__ __forceinline__ int dpp_i(int x) {
    return __builtin_amdgcn_mov_dpp(x, CTRL, 0xF, 0xF, false);
}
__device__ __forceinline__ float lane_f(float x, int l) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), l));
}
__device__ __forceinline__ int uni(int x) { return __builtin_amdgcn_readfirstlane(x); }

// DPP butterfly inside each 16-lane row (quad swaps, half-row and row mirrors), then the
// four row results combined through readlane.  Full wavefront active; every lane gets
// the result.
constexpr int kQuadSwap1 = 0xB1;   // quad_perm [1,0,3,2]
constexpr int kQuadSwap2 = 0x4E;   // quad_perm [2,3,0,1]
constexpr int kRowHalfMirror = 0x141;
constexpr int kRowMirror = 0x140;

__device__ __forceinline__ float wave_max(float x) {
    x = fmaxf(x, dpp<kQuadSwap1>(x));
    x = fmaxf(x, dpp<kQuadSwap2>(x));
    x = fmaxf(x, dpp<kRowHalfMirror>(x));
    x = fmaxf(x, dpp<kRowMirror>(x));
    return fmaxf(fmaxf(lane_f(x, 0), lane_f(x, 16)), fmaxf(lane_f(x, 32), lane_f(x, 48)));
}
__device__ __forceinline__ float wave_sum(float x) {
    x += dpp<kQuadSwap1>(x);
    x += dpp<kQuadSwap2>(x);
    x += dpp<kRowHalfMirror>(x);
    x += dpp<kRowMirror>(x);
    return (lane_f(x, 0) + lane_f(x, 16)) + (lane_f(x, 32) + lane_f(x, 48));
}

// (value, index) maximum: larger value wins, equal values go to the lower index.
__device__ __forceinline__ void take_better(float& v, int& i, float v2, int i2) {
    if (v2 > v || (v2 == v && i2 < i)) { v = v2; i = i2; }
}
template <int CTRL>
__device__ __forceinline__ void argmax_step(float& v, int& i) {
    const float v2 = dpp<CTRL>(v);
    const int i2 = dpp_i<CTRL>(i);
    take_better(v, i, v2, i2);
}
__device__ __forceinline__ void wave_argmax(float& v, int& i) {
    argmax_step<kQuadSwap1>(v, i);
    argmax_step<kQuadSwap2>(v, i);
    argmax_step<kRowHalfMirror>(v, i);
    argmax_step<kRowMirror>(v, i);
    float bv = lane_f(v, 0);
    int bi = __builtin_amdgcn_readlane(i, 0);
#pragma unroll
    for (int r = 16; r < 64; r += 16) take_better(bv, bi, lane_f(v, r), __builtin_amdgcn_readlane(i, r));
    v = bv;
    i = bi;
}

// The correctly rounded fp32 quotient v / s (fp32 v, s; s finite and nonzero) as the
// fp64 product of v with r = 1/s correctly rounded in fp64 (one fp64 division per
// 128-group), rounded once to fp32.  Where v / s is an fp32 normal it equals IEEE fp32
// division: a rounding boundary there is M = odd 25-bit integer * 2^c, v != M*s (the odd
// part of M*s has more than 24 bits), and v - M*s is a multiple of the grid 2^(b+c) of
// M*s (s = S*2^b) or of v's own grid, so v/s is more than 2^-49 * M away from every
// boundary, while the fp64 product is within 2^-52 of v/s.  Below the fp32 normal range
// the two may differ by one subnormal step; an E4M3 code does not see that (every
// |v/s| < 2^-10 encodes as a signed zero, sign kept by both).
__device__ __forceinline__ float quot_rn(float v, double r) { return (float)((double)v * r); }

// The quantiser scale amax / 448 rounded to fp32, for every fp32 amax: the quotient
// above with the constant reciprocal.  Here the argument extends below the normal range:
// 448 = 7*2^6 has three significant bits, so a boundary that amax/448 misses is more than
// 2^-27 away (relative), and where amax/448 is exactly a subnormal tie the product still
// lands on it (fp64 1/448 is within 2^-54, less than half an fp64 ulp of a value of at
// most 24 bits), so the final rounding sees the same tie.
__device__ __forceinline__ float e4m3_scale(float amax) { return quot_rn(amax, 1.0 / 448.0); }

// Two values -> two E4M3 codes (low byte first).  The hardware conversion rounds to
// nearest even but does not saturate, so magnitudes are clamped to 448 first.
__device__ __forceinline__ uint32_t e4m3x2(float a, float b) {
    a = fminf(fmaxf(a, -448.0f), 448.0f);
    b = fminf(fmaxf(b, -448.0f), 448.0f);
    return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false) & 0xFFFFu;
}

// Eight E4M3 codes (two dwords) -> eight fp16 values, exactly (every E4M3 value is an
// fp16 value; the conversion scale is 1).
__device__ __forceinline__ v8h e4m3x8_to_f16(uint32_t d0, uint32_t d1) {
    const v2h a = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8((int)d0, 1.0f, false);
    const v2h b = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8((int)d0, 1.0f, true);
    const v2h c = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8((int)d1, 1.0f, false);
    const v2h d = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8((int)d1, 1.0f, true);
    v8h r;
    r[0] = a[0]; r[1] = a[1]; r[2] = b[0]; r[3] = b[1];
    r[4] = c[0]; r[5] = c[1]; r[6] = d[0]; r[7] = d[1];
    return r;
}

// Operand layout of one 128-deep block (both MFMA operands use the same assignment, so
// their products pair up): lane l supplies row (A) or token column (B) l%16 and the
// bytes [16*(l/16), +16) and [64 + 16*(l/16), +16) of the block, held as two uint4.
// Each 16x16x32 fp16 MFMA takes 8 of those bytes per lane (sub-block s = 0..3 takes
// dwords 2s, 2s+1).  Result: lane l, element j = row 4*(l/16)+j, column l%16.
__device__ __forceinline__ v4f block_mma(const v4i& a0, const v4i& a1, const v4i& b0, const v4i& b1) {
    v4f c = {0.f, 0.f, 0.f, 0.f};
    c = __builtin_amdgcn_mfma_f32_16x16x32_f16(e4m3x8_to_f16(a0[0], a0[1]), e4m3x8_to_f16(b0[0], b0[1]), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x32_f16(e4m3x8_to_f16(a0[2], a0[3]), e4m3x8_to_f16(b0[2], b0[3]), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x32_f16(e4m3x8_to_f16(a1[0], a1[1]), e4m3x8_to_f16(b1[0], b1[1]), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x32_f16(e4m3x8_to_f16(a1[2], a1[3]), e4m3x8_to_f16(b1[2], b1[3]), c, 0, 0, 0);
    return c;
}

// block_mma with the A operand already decoded (a[i]: the fp16 values of sub-block i), for a
// weight block shared by several N tiles: the same products in the same order.
__device__ __forceinline__ v4f block_mma_a16(const v8h* a, const v4i& b0, const v4i& b1) {
    v4f c = {0.f, 0.f, 0.f, 0.f};
    c = __builtin_amdgcn_mfma_f32_16x16x32_f16(a[0], e4m3x8_to_f16(b0[0], b0[1]), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x32_f16(a[1], e4m3x8_to_f16(b0[2], b0[3]), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x32_f16(a[2], e4m3x8_to_f16(b1[0], b1[1]), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x32_f16(a[3], e4m3x8_to_f16(b1[2], b1[3]), c, 0, 0, 0);
    return c;
}

// The same 128-deep block contracted by one e4m3 x e4m3 MFMA (16x16x128, both operands
// OCP E4M3, block scales 2^0) in the operand layout above: each lane's 32 bytes are its
// eight dwords, in the same K order in A and B, so the products pair up as in block_mma.
// Its block sums carry a relative error of about 2^-15 (measured), so it serves only the
// down projection, whose block sums are scaled and accumulated but never requantised.
typedef int v8i __attribute__((ext_vector_type(8)));
constexpr int kMfmaFmtE4M3 = 0;
constexpr int kMfmaScaleOne = 127;   // E8M0 exponent of 1.0
__device__ __forceinline__ v4f block_mma_f8(const v4i& a0, const v4i& a1, const v4i& b0, const v4i& b1) {
    const v8i a = {a0[0], a0[1], a0[2], a0[3], a1[0], a1[1], a1[2], a1[3]};
    const v8i b = {b0[0], b0[1], b0[2], b0[3], b1[0], b1[1], b1[2], b1[3]};
    const v4f z = {0.f, 0.f, 0.f, 0.f};
    return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, z, kMfmaFmtE4M3, kMfmaFmtE4M3, 0, kMfmaScaleOne, 0,
                                                            kMfmaScaleOne);
}

// Bounded wait until *p >= target on an LDS flag; false on abort or timeout.  Inlined where
// a translation unit asks for it (a call from a streaming loop costs a register save and
// restore around it); a call elsewhere.
#ifndef MONOMOE_WAIT_INLINE
#define MONOMOE_WAIT_INLINE
#endif
static __device__ MONOMOE_WAIT_INLINE bool wait_lds(const int* p, int target, const int* abort_flag, uint64_t limit) {
    if (lds_ld(p) >= target) {
        compiler_fence();   // the data the flag guards is read after it
        return true;
    }
    const uint64_t t0 = now();
    while (true) {
        if (lds_ld(p) >= target) {
            compiler_fence();
            return true;
        }
        if (lds_ld(abort_flag)) return false;
        if (now() - t0 > limit) return false;
        __builtin_amdgcn_s_sleep(1);
    }
}

// ------------------------------------------------------------------------------------
// routing helpers
// ------------------------------------------------------------------------------------
// Maximum over each 16-lane row (quad swaps, half-row and row mirrors); every lane of the
// row gets its row's maximum.
__device__ __forceinline__ float row16_max(float x) {
    x = fmaxf(x, dpp<kQuadSwap1>(x));
    x = fmaxf(x, dpp<kQuadSwap2>(x));
    x = fmaxf(x, dpp<kRowHalfMirror>(x));
    return fmaxf(x, dpp<kRowMirror>(x));
}

// Block-wise FP8 quantisation of the whole input [T,H] into LDS (row pitch H+16 bytes,
// then the fp32 scales [T,H/128]).  Sixteen lanes (one DPP row) own one 128-element
// group, eight values each: s = amax/448 and codes = e4m3(v/s) with the fp32 quotient
// (quot_rn), the same arithmetic as every other quantisation in this file.  Scale rows
// T..kTMax-1 are zeroed.  Threads 0 .. NTH-1 take part (all of the workgroup by default).
template <int H, int NTH = kThreads>
__device__ __forceinline__ void quantise_input(const uint16_t* __restrict__ x, int T, uint8_t* xq_s, float* xs_s,
                                               int tid, uint8_t* d_xq, float* d_xs) {
    constexpr int HB = H / 128, XROW = H + 16, CPR = H / 8, UNR = 4;
    constexpr int kThreads = NTH;   // the threads taking part: tid in [0, NTH)
    const int nch = T * CPR;   // a multiple of 16, so DPP rows are all valid or all not
    for (int c0 = 0; c0 < nch; c0 += UNR * kThreads) {
        // All loads of a pass are issued back to back (clamped addresses, no branches in
        // between, so none waits for another); slices u with c0 + u * kThreads >= nch hold
        // no chunk of any thread and skip their arithmetic (a uniform branch).
        uint4 v[UNR];
#pragma unroll
        for (int u = 0; u < UNR; ++u)
            v[u] = *reinterpret_cast<const uint4*>(x + (size_t)min(c0 + u * kThreads + tid, nch - 1) * 8);
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            if (c0 + u * kThreads >= nch) break;
            const int c = c0 + u * kThreads + tid;
            const uint32_t w4[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
            float f[8];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                f[2 * q] = bf16_to_f32(w4[q] & 0xFFFFu);
                f[2 * q + 1] = bf16_to_f32(w4[q] >> 16);
            }
            float a = 0.0f;
#pragma unroll
            for (int q = 0; q < 8; ++q) a = fmaxf(a, fabsf(f[q]));
            const float amax = row16_max(a);
            float sc = e4m3_scale(amax);
            uint32_t d0 = 0u, d1 = 0u;
            if (amax == 0.0f || sc == 0.0f) {
                sc = 0.0f;
            } else {
                const double r = 1.0 / (double)sc;
                d0 = e4m3x2(quot_rn(f[0], r), quot_rn(f[1], r)) | (e4m3x2(quot_rn(f[2], r), quot_rn(f[3], r)) << 16);
                d1 = e4m3x2(quot_rn(f[4], r), quot_rn(f[5], r)) | (e4m3x2(quot_rn(f[6], r), quot_rn(f[7], r)) << 16);
            }
            if (c < nch) {
                const int t = c / CPR, o = (c - t * CPR) * 8;
                *reinterpret_cast<uint2*>(xq_s + t * XROW + o) = make_uint2(d0, d1);
                if ((tid & 15) == 0) xs_s[t * HB + o / 128] = sc;
                if (d_xq) {
                    *reinterpret_cast<uint2*>(d_xq + (size_t)t * H + o) = make_uint2(d0, d1);
                    if ((tid & 15) == 0) d_xs[t * HB + o / 128] = sc;
                }
            }
        }
    }
    for (int i = T * HB + tid; i < kTMax * HB; i += kThreads) xs_s[i] = 0.0f;
}

// Quantised-input exchange, used when the input is large (more than kLocalQuantChunks
// 8-element chunks per thread; below that the replicated quantisation is cheaper than
// the extra round trip, measured): instead of every workgroup quantising the whole input,
// the 128-groups are split over the workgroups; each quantises its share once (the same
// arithmetic as quantise_loaded) and publishes the codes as tagged words {4 codes, tag}
// and the scales as {fp32, tag}; every workgroup then polls all of them into its LDS.
template <int H>
__device__ __forceinline__ void publish_input_groups(const KParams& p, int T, int wg, int G, int tid, uint32_t tag) {
    constexpr int HB = H / 128, GPP = kThreads / 16;   // groups per pass: one per DPP row
    const int NG = T * HB;
    const int q0 = range_lo(wg, G, NG);
    const int q1 = range_lo(wg + 1, G, NG);
    const uint64_t tag_hi = (uint64_t)tag << 32;
    const int r = tid & 15;
    for (int qb = q0; qb < q1; qb += GPP) {
        if (qb + 4 * (tid >> 6) >= q1) break;   // no group for this wavefront (uniform)
        const int q = qb + (tid >> 4);
        const int qq = min(q, q1 - 1);          // rows past the end repeat the last group
        const int t = qq / HB, g = qq - t * HB, o = g * 128 + 8 * r;
        const uint4 v = *reinterpret_cast<const uint4*>(p.x + (size_t)t * H + o);
        const uint32_t w4[4] = {v.x, v.y, v.z, v.w};
        float f[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            f[2 * i] = bf16_to_f32(w4[i] & 0xFFFFu);
            f[2 * i + 1] = bf16_to_f32(w4[i] >> 16);
        }
        float a = 0.0f;
#pragma unroll
        for (int i = 0; i < 8; ++i) a = fmaxf(a, fabsf(f[i]));
        const float amax = row16_max(a);
        float sc = e4m3_scale(amax);
        uint32_t d0 = 0u, d1 = 0u;
        if (amax == 0.0f || sc == 0.0f) {
            sc = 0.0f;
        } else {
            const double rc = 1.0 / (double)sc;
            d0 = e4m3x2(quot_rn(f[0], rc), quot_rn(f[1], rc)) | (e4m3x2(quot_rn(f[2], rc), quot_rn(f[3], rc)) << 16);
            d1 = e4m3x2(quot_rn(f[4], rc), quot_rn(f[5], rc)) | (e4m3x2(quot_rn(f[6], rc), quot_rn(f[7], rc)) << 16);
        }
        if (q < q1) {
            const size_t wi = ((size_t)t * H + o) / 4;
            st_co(p.xqw + wi, tag_hi | d0);
            st_co(p.xqw + wi + 1, tag_hi | d1);
            if (r == 0) st_co(p.xsw + (size_t)t * HB + g, tag_hi | __float_as_uint(sc));
            if (p.d_xq) {
                *reinterpret_cast<uint2*>(p.d_xq + (size_t)t * H + o) = make_uint2(d0, d1);
                if (r == 0) p.d_xs[t * HB + g] = sc;
            }
        }
    }
}

// Every workgroup's copy of the published quantised input: polls the tagged code and
// scale words into LDS (rows of pitch H+16, then the scales; rows T..kTMax-1 of the
// scales zeroed), in batches of B 16-byte pairs per thread.  False on timeout or when
// another workgroup has recorded an error.
template <int H>
__device__ __forceinline__ bool fetch_input(const KParams& p, int T, uint8_t* xq_s, float* xs_s, int tid, uint32_t tag,
                                            uint32_t* status, uint64_t limit) {
    constexpr int HB = H / 128, XROW = H + 16, B = 8;
    const int npair = T * H / 8;   // a pair: two words, eight codes
    const __amdgpu_buffer_rsrc_t rq = buf_rsrc(p.xqw);
    const uint64_t t0 = now();
    for (int base = 0; base < npair; base += B * kThreads) {
        v4i d[B];
        while (true) {
            bool fresh = true;
#pragma unroll
            for (int b = 0; b < B; ++b) {
                const int i = min(base + b * kThreads + tid, npair - 1);
                d[b] = ld_co16(rq, (uint32_t)i * 16u);
            }
#pragma unroll
            for (int b = 0; b < B; ++b) fresh = fresh && (uint32_t)d[b][1] == tag && (uint32_t)d[b][3] == tag;
            if (__ballot(!fresh) == 0) break;
            if (ld_co(status) != kDevOk) return false;
            if (now() - t0 > limit) {
                set_status(status, kDevTimeout);
                return false;
            }
            __builtin_amdgcn_s_sleep(1);
        }
#pragma unroll
        for (int b = 0; b < B; ++b) {
            const int i = base + b * kThreads + tid;
            if (i < npair) {
                const int t = (8 * i) / H, o = 8 * i - t * H;
                *reinterpret_cast<uint2*>(xq_s + t * XROW + o) = make_uint2((uint32_t)d[b][0], (uint32_t)d[b][2]);
            }
        }
    }
    for (int i = tid; i < kTMax * HB; i += kThreads) {
        float v = 0.0f;
        if (i < T * HB) {
            while (true) {
                const uint64_t w = ld_co(p.xsw + i);
                if ((uint32_t)(w >> 32) == tag) {
                    v = __uint_as_float((uint32_t)w);
                    break;
                }
                if (ld_co(status) != kDevOk) return false;
                if (now() - t0 > limit) {
                    set_status(status, kDevTimeout);
                    return false;
                }
                __builtin_amdgcn_s_sleep(1);
            }
        }
        xs_s[i] = v;
    }
    return true;
}

// Wavefront maximum delivered to every lane: the row butterfly, then the GFX9 row
// broadcasts (lane 15 of each row into the next row, lane 31 into rows 2 and 3) leave
// the total in lane 63.
__device__ __forceinline__ float row_bcast_max(float x, int ctrl_is_31) {
    const int xi = __float_as_int(x);
    const int y = ctrl_is_31 ? __builtin_amdgcn_update_dpp(xi, xi, 0x143, 0xC, 0xF, false)
                             : __builtin_amdgcn_update_dpp(xi, xi, 0x142, 0xA, 0xF, false);
    return fmaxf(x, __int_as_float(y));
}
__device__ __forceinline__ float wave_max_all(float x) {
    x = row16_max(x);
    x = row_bcast_max(x, 0);
    x = row_bcast_max(x, 1);
    return lane_f(x, 63);
}

// Integer wavefront maximum delivered as a scalar: the same butterfly and row
// broadcasts, each step a single DPP-fused integer maximum.
__device__ __forceinline__ int wave_max_i32(int x) {
    x = max(x, dpp_i<kQuadSwap1>(x));
    x = max(x, dpp_i<kQuadSwap2>(x));
    x = max(x, dpp_i<kRowHalfMirror>(x));
    x = max(x, dpp_i<kRowMirror>(x));
    x = max(x, __builtin_amdgcn_update_dpp(x, x, 0x142, 0xA, 0xF, false));
    x = max(x, __builtin_amdgcn_update_dpp(x, x, 0x143, 0xC, 0xF, false));
    return __builtin_amdgcn_readlane(x, 63);
}

// Top-k of NT tokens' router logits by one wavefront, the tokens interleaved so that
// their dependency chains overlap (softmax routing with top-k, Sec. 4.1; the softmax is
// monotone, so selecting on logits is selecting on probabilities): k rounds of "largest
// remaining logit, lower expert index on ties".  Lane l holds experts l + 64 i, i < EPL.
// The winner of a round is found with a value maximum followed by ballots of the lanes
// that hold it, so no round branches per lane.  Writes ids[n][0..k) (LDS; ids[n] ==
// nullptr skips token n); an expert that cannot be determined (NaN logits) is reported
// as -1.  The routing weights are computed later, by routing_weights.  The logits are tagged words: the wavefront polls until
// every word carries this launch's tag (false on timeout or when another workgroup has
// recorded an error).  With `publish` (an LDS counter; one token), each round's selection is
// also written to ids[0][j] at once and the counter raised to j + 1, so consumers of the
// first selections need not wait for the last.
template <int EPL, int NT>
__device__ __forceinline__ bool topk_tokens(const uint64_t* const* rows, int E, int K, int lane,
                                            uint32_t tag, uint32_t* status, uint64_t limit, int* const* ids,
                                            int policy, const float* sel_bias, uint64_t* st_logits,
                                            uint64_t* st_selected, int* publish = nullptr) {
    float lv[NT][EPL];
    float bias[EPL];   // expert-selection bias of sigmoid routing
#pragma unroll
    for (int i = 0; i < EPL; ++i) bias[i] = sel_bias ? sel_bias[min(lane + 64 * i, E - 1)] : 0.0f;
    {
        const uint64_t t0 = now();
        while (true) {
            uint64_t raw[NT][EPL];
#pragma unroll
            for (int n = 0; n < NT; ++n)
#pragma unroll
                for (int i = 0; i < EPL; ++i) raw[n][i] = ld_co(rows[n] + min(lane + 64 * i, E - 1));
            bool fresh = true;
#pragma unroll
            for (int n = 0; n < NT; ++n)
#pragma unroll
                for (int i = 0; i < EPL; ++i) {
                    fresh = fresh && (uint32_t)(raw[n][i] >> 32) == tag;
                    lv[n][i] = __uint_as_float((uint32_t)raw[n][i]);
                }
            if (__ballot(!fresh) == 0) break;
            if (ld_co(status) != kDevOk) return false;
            if (now() - t0 > limit) {
                set_status(status, kDevTimeout);
                return false;
            }
            __builtin_amdgcn_s_sleep(1);
        }
    }
    if (st_logits && lane == 0) *st_logits = now();
    if (policy == kRouteSigmoidBias) {   // rank by logistic(logit) + selection bias
#pragma unroll
        for (int n = 0; n < NT; ++n)
#pragma unroll
            for (int i = 0; i < EPL; ++i) lv[n][i] = 1.0f / (1.0f + expf(-lv[n][i])) + bias[i];
    }
    // Selection on order-preserving integer keys of the scores (one integer maximum per
    // DPP step, no NaN canonicalisation): key(v) is monotonic in v; -0 is folded into +0
    // and NaN, padding and taken experts get INT_MIN.
    int key[NT][EPL];
#pragma unroll
    for (int n = 0; n < NT; ++n)
#pragma unroll
        for (int i = 0; i < EPL; ++i) {
            const float f = lv[n][i] + 0.0f;
            const int bits = __float_as_int(f);
            key[n][i] = (lane + 64 * i < E && f == f) ? (bits ^ ((bits >> 31) & 0x7FFFFFFF)) : INT_MIN;
        }
    int my_key[NT], my_id[NT];
#pragma unroll
    for (int n = 0; n < NT; ++n) {
        my_key[n] = INT_MIN;
        my_id[n] = -1;
    }
    for (int j = 0; j < K; ++j) {
#pragma unroll
        for (int n = 0; n < NT; ++n) {
            int lm = key[n][0];
#pragma unroll
            for (int i = 1; i < EPL; ++i) lm = max(lm, key[n][i]);
            const int bk = wave_max_i32(lm);
            int bi = -1;
#pragma unroll
            for (int i = EPL - 1; i >= 0; --i) {
                const uint64_t b = __ballot(key[n][i] == bk);
                bi = b ? 64 * i + (int)__builtin_ctzll(b) : bi;
            }
            bi = uni(bi);
#pragma unroll
            for (int i = 0; i < EPL; ++i) key[n][i] = (lane + 64 * i == bi) ? INT_MIN : key[n][i];
            if (lane == j) {
                my_key[n] = bk;
                my_id[n] = bi;
            }
            if (publish != nullptr && n == 0 && lane == 0) {   // this round's selection, at once
                ids[0][j] = bi;
                lds_st(publish, j + 1);
            }
        }
    }
#pragma unroll
    for (int n = 0; n < NT; ++n)
        if (ids[n] != nullptr && lane < K) ids[n][lane] = my_id[n];
    if (st_selected && lane == 0 && my_key[0] != INT_MIN) *st_selected = now();
    return true;
}

// Routing weights of every token (Sec. 4.1), from the selection in ids [T,k] and the
// tagged logits (already complete).  Softmax routing: with m the token's largest logit
// (its first selected expert), w_j = exp(l_j - m) / (sum of exp(l - m) over the
// selection, in selection order) when renormalised, else / (the same sum over all E
// experts).  Sigmoid routing: w_j = scale * a_j / (sum of the selected a, in selection
// order), a = 1/(1+exp(-l)).  One wavefront; pair p = t*k + j is handled in slot p / 64 of
// lane p mod 64 (T*k <= 64*NS).  w doubles as the LDS scratch; every pass reads all it needs
// before any lane overwrites it.  An undetermined expert (-1) gets weight 0.
template <int NS>
__device__ __forceinline__ void routing_weights(const uint64_t* logits, const int* ids, float* w, int T, int E,
                                                int K, int renorm, int policy, float scale, int lane) {
    const bool sig = policy == kRouteSigmoidBias;
    const int np = T * K;
    float v[NS];
#pragma unroll
    for (int r = 0; r < NS; ++r) {   // selected logits -> w
        const int pr = 64 * r + lane;
        v[r] = 0.0f;
        if (pr < np) {
            const int e = ids[pr];
            if (e >= 0 && e < E) v[r] = __uint_as_float((uint32_t)ld_co(logits + (size_t)(pr / K) * E + e));
        }
    }
#pragma unroll
    for (int r = 0; r < NS; ++r)
        if (64 * r + lane < np) w[64 * r + lane] = v[r];
    lgkm_drain();
#pragma unroll
    for (int r = 0; r < NS; ++r) {   // exp(l - m), m from the token's first pair; or a(l)
        const int pr = 64 * r + lane;
        if (pr < np) {
            const int e = ids[pr];
            const float u = sig ? 1.0f / (1.0f + expf(-v[r])) : expf(v[r] - w[(pr / K) * K]);
            v[r] = (e >= 0 && e < E) ? u : 0.0f;
        }
    }
    lgkm_drain();
#pragma unroll
    for (int r = 0; r < NS; ++r)
        if (64 * r + lane < np) w[64 * r + lane] = v[r];
    lgkm_drain();
    float den[NS];
    if (renorm || sig) {
#pragma unroll
        for (int r = 0; r < NS; ++r) {
            const int pr = 64 * r + lane;
            den[r] = 1.0f;
            if (pr < np) {
                float sum = 0.0f;
                for (int j = 0; j < K; ++j) sum += w[(pr / K) * K + j];
                den[r] = sum;
            }
        }
    } else {
#pragma unroll
        for (int r = 0; r < NS; ++r) den[r] = 1.0f;
        for (int t = 0; t < T; ++t) {
            const int e0 = ids[t * K];
            const float m = __uint_as_float((uint32_t)ld_co(logits + (size_t)t * E + ((e0 >= 0 && e0 < E) ? e0 : 0)));
            float se = 0.0f;
            for (int e = lane; e < E; e += 64) se += expf(__uint_as_float((uint32_t)ld_co(logits + (size_t)t * E + e)) - m);
            const float tot = wave_sum(se);
#pragma unroll
            for (int r = 0; r < NS; ++r)
                if (64 * r + lane < np && (64 * r + lane) / K == t) den[r] = tot;
        }
    }
    lgkm_drain();
    const float mul = sig ? scale : 1.0f;
#pragma unroll
    for (int r = 0; r < NS; ++r)
        if (64 * r + lane < np) w[64 * r + lane] = mul * (v[r] / den[r]);
    lgkm_drain();
}

// topk_tokens with the experts-per-lane count specialised on E (E <= kEMax).
template <int NT>
__device__ __forceinline__ bool topk_bucket(const uint64_t* const* rows, int E, int K, int lane, uint32_t tag,
                                            uint32_t* status, uint64_t limit, int* const* ids, int policy,
                                            const float* sel_bias, uint64_t* stl, uint64_t* sts,
                                            int* publish = nullptr) {
    if (E <= 64) return topk_tokens<1, NT>(rows, E, K, lane, tag, status, limit, ids, policy, sel_bias, stl, sts, publish);
    if (E <= 128) return topk_tokens<2, NT>(rows, E, K, lane, tag, status, limit, ids, policy, sel_bias, stl, sts, publish);
    if (E <= 256) return topk_tokens<4, NT>(rows, E, K, lane, tag, status, limit, ids, policy, sel_bias, stl, sts, publish);
    return topk_tokens<8, NT>(rows, E, K, lane, tag, status, limit, ids, policy, sel_bias, stl, sts, publish);
}

// Router logits of experts wg, wg + G, ... (Sec. 4.1): the bf16 dot product of each
// token row with each router row, accumulated in fp32 (per thread over its 8-element
// chunks, then over the workgroup), plus the optional bias, stored as tagged words.  NT
// is the token bucket (T <= NT): the token loop is unrolled to NT, rows beyond T are
// clamped loads whose sums are dropped.
template <int H, int NT>
__device__ __forceinline__ void router_rows(const KParams& p, int wg, int G, int tid, uint32_t tag, float* red) {
    const int T = p.T, E = p.E;
    const int lane = tid & 63, wv = tid >> 6;
    for (int e = wg; e < E; e += G) {
        float acc_t[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) acc_t[t] = 0.0f;
        const uint16_t* rrow = p.rw + (size_t)e * H;
        for (int c = tid; c < H / 8; c += kThreads) {
            // all loads first (token index clamped, so the count is fixed), then the FMAs
            const uint4 rv = *reinterpret_cast<const uint4*>(rrow + c * 8);
            uint4 xv[NT];
#pragma unroll
            for (int t = 0; t < NT; ++t)
                xv[t] = *reinterpret_cast<const uint4*>(p.x + (size_t)min(t, T - 1) * H + c * 8);
            const uint32_t rw4[4] = {rv.x, rv.y, rv.z, rv.w};
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const uint32_t x4[4] = {xv[t].x, xv[t].y, xv[t].z, xv[t].w};
                float a = acc_t[t];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    a = fmaf(bf16_to_f32(x4[q] & 0xFFFFu), bf16_to_f32(rw4[q] & 0xFFFFu), a);
                    a = fmaf(bf16_to_f32(x4[q] >> 16), bf16_to_f32(rw4[q] >> 16), a);
                }
                acc_t[t] = a;
            }
        }
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            if (t < T) {
                const float s = wave_sum(acc_t[t]);
                if (lane == 0) red[wv * kTMax + t] = s;
            }
        }
        __syncthreads();
        if (tid < T) {
            float s = 0.0f;
            for (int v = 0; v < kWaves; ++v) s += red[v * kTMax + tid];
            if (p.bias) s += p.bias[e];
            st_co(p.logits + (size_t)tid * E + e, ((uint64_t)tag << 32) | __float_as_uint(s));
        }
        __syncthreads();
    }
}
// Router logits of one expert e for the token rows x[0..T) (a chunk of a larger input),
// stored into logits[t*E + e]: the same arithmetic as router_rows.  All threads of the
// workgroup take part.
template <int H, int NT>
__device__ __forceinline__ void router_row_of(const KParams& p, int e, const uint16_t* x, int T, uint64_t* logits,
                                              int tid, uint32_t tag, float* red) {
    const int E = p.E;
    const int lane = tid & 63, wv = tid >> 6;
    float acc_t[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) acc_t[t] = 0.0f;
    const uint16_t* rrow = p.rw + (size_t)e * H;
    for (int c = tid; c < H / 8; c += kThreads) {
        const uint4 rv = *reinterpret_cast<const uint4*>(rrow + c * 8);
        uint4 xv[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t)
            xv[t] = *reinterpret_cast<const uint4*>(x + (size_t)min(t, T - 1) * H + c * 8);
        const uint32_t rw4[4] = {rv.x, rv.y, rv.z, rv.w};
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const uint32_t x4[4] = {xv[t].x, xv[t].y, xv[t].z, xv[t].w};
            float a = acc_t[t];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                a = fmaf(bf16_to_f32(x4[q] & 0xFFFFu), bf16_to_f32(rw4[q] & 0xFFFFu), a);
                a = fmaf(bf16_to_f32(x4[q] >> 16), bf16_to_f32(rw4[q] >> 16), a);
            }
            acc_t[t] = a;
        }
    }
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        if (t < T) {
            const float s = wave_sum(acc_t[t]);
            if (lane == 0) red[wv * kTMax + t] = s;
        }
    }
    __syncthreads();
    if (tid < T) {
        float s = 0.0f;
        for (int v = 0; v < kWaves; ++v) s += red[v * kTMax + tid];
        if (p.bias) s += p.bias[e];
        st_co(logits + (size_t)tid * E + e, ((uint64_t)tag << 32) | __float_as_uint(s));
    }
    __syncthreads();
}

}  // namespace monomoe
