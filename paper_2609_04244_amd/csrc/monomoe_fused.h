// Persistent, weight-major fused routed-MoE decode kernel for gfx950 (MI355X).
//
// One launch computes the whole routed-MoE operator of MonoMoE (arXiv 2609.04244,
// Sec. 3): router logits, softmax/top-k, per-128-group E4M3 input quantisation,
// block-FP8 gate/up projection, SiLU(gate)*up, requantisation, block-FP8 down
// projection and the top-k weighted reduction.
//
// Decomposition (Sec. 3.1, Eq. 9).  Workgroups are partitioned over EXPERT-WEIGHT tiles,
// never over token tiles.  A gate/up unit is 8 gate rows plus the 8 matching up rows of
// one active expert; a down unit is 16 output rows of one active expert.  Each unit is a
// 16-row MFMA M tile and the whole decode token tile (T <= 16) is the MFMA N side; the
// K dimension of a unit is split over the compute wavefronts of the workgroup in
// 128-deep blocks.  Every 128-deep block is one fp32 MFMA block sum to which the fp32
// weight block scale and the token's activation group scale are applied.
//
// Numerics.  Weights and activations stay E4M3 in HBM and LDS.  In the gate/up
// projection each 128-deep block is decoded exactly to fp16 in registers and contracted
// with four 16x16x32 fp16 MFMAs chained in fp32: the 8-bit MFMA forms accumulate a
// 128-deep block with roughly 2^-15 relative error, enough to flip requantised E4M3 codes
// of the SwiGLU output, while fp16 inputs give correctly rounded fp32 block sums in
// practice.  The down projection's block sums are never requantised, so there each block
// is one 16x16x128 e4m3 MFMA on the codes as loaded.
//
// Wavefront roles (Sec. 3.3, warp specialisation, re-cast for CDNA).  Four compute
// wavefronts (one per SIMD) only stream weights (dwordx4 loads into a register ring that
// stays full across unit boundaries and from the gate/up into the down projection) and
// run MFMAs; each writes its partial sums of a unit into an LDS hand-off slot.  The helper
// wavefront does everything that would otherwise stall the weight stream: the gate/up
// epilogue (SiLU(gate)*up and its store), the per-128-group requantisation of the next
// expert's activation into LDS and the down epilogue (routing weight, contribution
// store).  Where a down unit is computed by one wavefront alone (I < 1024: fewer 256-deep
// tasks per unit than wavefronts), that wavefront applies the routing weight and stores the
// contribution itself, and publishes its progress so that the helper knows when an
// activation buffer is free again.
//
// Synchronisation (Sec. 3.2, readiness-based hand-off).  Data that crosses workgroups
// is written as 8-byte words {fp32 value, launch tag} with single-copy-atomic sc1
// stores, so a consumer polls the data itself: a word whose tag equals this launch's tag
// is final.  This replaces "store, wait for the store to complete, bump a counter, poll
// the counter, load the data" by "store; poll-load", and needs no counter resets between
// launches (each workgroup keeps a launch epoch; all epochs advance in lockstep).  Router
// logits (all top-k computations depend on every router row), SiLU activations (a down
// unit depends on every gate/up unit of its expert) and the routing-weighted expert
// outputs travel this way.  Every 16-column output tile has one designated reducer
// reduction that sums a token's k contributions in top-k order, so the output does not
// depend on timing.  Cross-XCD coherence comes from the sc1 policy of the tagged
// accesses; no L2 writeback or invalidate fence is used.  Every wait is bounded by
// s_memrealtime; on expiry the kernel records a status word and drains.  The grid never
// exceeds one workgroup per CU (the host checks occupancy), so every workgroup a wait
// depends on is resident.
//
// This header holds the kernel template (monomoe_fused<H, I, RING, ONE>); it is instantiated
// by monomoe_kernel.hip (the general kernel, ONE = false, and the compiled-shape table) and by
// monomoe_kernel_one.hip (the one-token specialisation, ONE = true), two translation units so
// that each one's code generation sees only its own kernels.
#pragma once

#include "monomoe_device.h"

// Inlining of the weight-load cursor's helpers (lbase, lnext, ranked): forced by the
// translation units of the kernel (a call from the streaming loop spills the weight ring
// to scratch); left to the compiler elsewhere.
#ifndef MONOMOE_CURSOR_INLINE
#define MONOMOE_CURSOR_INLINE
#endif

namespace monomoe {

// Outputs o0 .. o0+63 of output tile ht (16 columns; output o is token o / 16, column
// o % 16): the sum of each token's k tagged contributions contrib[t*k + j][ht*16 + col]
// over j in top-k order, polled until all carry this launch's tag, then rounded to bf16
// (the fp32 sum also goes to the test hook).  One wavefront, lane l owns output o0 + l.
// False on timeout or when another workgroup has recorded an error.
// (Always inlined: a call would pass the kernel's argument block through scratch memory.)
template <int H>
__device__ __attribute__((always_inline)) bool reduce_chunk(const KParams& p, int ht, int o0, int T, int K, uint32_t tag, int lane,
                             uint32_t* status, uint64_t limit) {
    const uint64_t t0 = now();
    const int o = min(o0 + lane, T * 16 - 1);
    const int t = o >> 4, col = o & 15;
    const uint64_t* src = p.contrib + (size_t)t * K * H + ht * 16 + col;
    float sum;
    while (true) {
        uint64_t v[kKMax];
#pragma unroll
        for (int j = 0; j < kKMax; ++j) v[j] = (j < K) ? ld_co(src + (size_t)j * H) : 0ull;
        bool fresh = true;
        sum = 0.0f;
#pragma unroll
        for (int j = 0; j < kKMax; ++j) {
            if (j < K) {
                fresh = fresh && (uint32_t)(v[j] >> 32) == tag;
                sum += __uint_as_float((uint32_t)v[j]);
            }
        }
        if (__ballot(!fresh) == 0) break;
        if (ld_co(status) != kDevOk) return false;
        if (now() - t0 > limit) {
            set_status(status, kDevTimeout);
            return false;
        }
        __builtin_amdgcn_s_sleep(1);
    }
    if (o0 + lane < T * 16) {
        p.out[(size_t)t * H + ht * 16 + col] = f32_to_bf16(sum);
        if (p.d_out) p.d_out[(size_t)t * H + ht * 16 + col] = sum;
    }
    return true;
}

// ------------------------------------------------------------------------------------
// the kernel
// ------------------------------------------------------------------------------------
template <int H, int I, int RING, bool ONE>
__global__ __launch_bounds__(kThreads) void monomoe_fused(const KParams p) {
    constexpr int HB = H / 128;           // K blocks of the gate/up projection
    constexpr int IB = I / 128;           // K blocks of the down projection
    constexpr int UPE = I / 8;            // gate/up units per expert
    constexpr int DNE = H / 16;           // down units per expert (= 16-row output tiles)
    constexpr int XROW = H + 16;          // LDS row pitch of the quantised input
    constexpr int AROW = I + 16;          // LDS row pitch of the requantised act
    constexpr int NC = kComputeWaves;
    constexpr int HP = HB / 2;            // 256-deep tasks (block pairs) of a gate/up unit
    constexpr int IP = IB / 2;            // ... of a down unit
    // A phase whose units have at least NC tasks deals tasks round-robin over the compute
    // wavefronts (every wave contributes to every unit); a phase with fewer tasks per unit
    // deals whole units round-robin (one contributor per unit, so no wave runs one task
    // per unit hand-off).
    constexpr int NCU = HP < NC ? 1 : NC;    // wavefronts contributing to a gate/up unit
    constexpr int NCD = IP < NC ? 1 : NC;    // ... to a down unit
    static_assert(HB % 2 == 0 && IB % 2 == 0, "tasks are pairs of 128-deep blocks");

    extern __shared__ __align__(16) uint8_t lds_dyn[];
    __shared__ float red[kWaves * kTMax];
    __shared__ int sel_ids[kTMax * kKMax];
    __shared__ float sel_w[kTMax * kKMax];
    __shared__ uint32_t emask[kEMax];
    __shared__ int act_e[kUMax];
    __shared__ uint32_t act_m[kUMax];
    __shared__ uint8_t act_j[kUMax * kTMax];   // [u][t]: top-k position of expert slot u in token t
    __shared__ int h_pi[kTMax], h_t[kTMax];     // helper scratch: routed tokens of one expert
    __shared__ int s_U, s_fail;
    __shared__ int f_abort, f_consumed;
    __shared__ int f_cnt[kSlotsMax];
    __shared__ int f_aq_seq[2];
    __shared__ int f_dn_prog[kComputeWaves];   // direct down epilogues: each wave's next unfinished down unit
    __shared__ int f_rank, f_xq;                // one-token path: selections published, input quantised

    const int T = ONE ? 1 : p.T, E = p.E, K = p.k;   // ONE: the one-token specialisation
    const int G = gridDim.x, wg = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63, wv = uni(tid >> 6);
    uint32_t* ctl = p.ctl;
    uint32_t* status = ctl + kCtlStatus;
    const uint64_t limit = p.spin_limit;
    // this launch's tag: the workgroup's completed-launch count + 1 (the same in every
    // workgroup, since all of them complete every launch)
    const uint32_t tag = ld_co(ctl + kCtlEpoch + wg) + 1u;

    const int naq = p.naq;
    const int smask = p.nslots - 1;   // slot of hand-off sequence number q: q & smask
    const int aq_bytes = lds_aq_buffer_bytes(I, T);   // one requantised-act buffer
    uint8_t* xq_s = lds_dyn;
    float* xs_s = reinterpret_cast<float*>(lds_dyn + T * XROW);
    v4f* part = reinterpret_cast<v4f*>(lds_dyn + lds_region_bytes(H, I, T, naq));

    if (tid == 0) {
        s_fail = 0;
        f_abort = 0;
        f_consumed = 0;
        f_aq_seq[0] = 0;
        f_aq_seq[1] = 0;
        f_rank = 0;
        f_xq = 0;
    }
    if (tid < kSlotsMax) f_cnt[tid] = 0;
    if (tid < kComputeWaves) f_dn_prog[tid] = tid;   // a wave's first down unit (whole units dealt round-robin)
    for (int e = tid; e < E; e += kThreads) emask[e] = 0u;
    // the flags are set before any wavefront uses them (workgroups without router rows have
    // no other barrier before their first flag accesses)
    __syncthreads();
    if (tid == 0) stamp(p.stamps, wg, kStEntry);
    MONOMOE_PERTURB(0, 0);

    // ---------------- stage 0: router slice + input quantisation slice ----------------
    // A large input is quantised once, split over the workgroups, and exchanged (see below);
    // each workgroup publishes its share first, so that the shares travel while the router
    // rows are computed.
    const bool xq_exchange = !ONE && T * (H / 8) > kLocalQuantChunks * kThreads;
    static_assert(4 * (H / 8) <= kLocalQuantChunks * kThreads, "the input exchange starts above four tokens");
    if (ONE || T == 1) router_rows<H, 1>(p, wg, G, tid, tag, red);
    else if (T == 2) router_rows<H, 2>(p, wg, G, tid, tag, red);
    else if (T <= 4) router_rows<H, 4>(p, wg, G, tid, tag, red);
    else {
        if (xq_exchange) publish_input_groups<H>(p, T, wg, G, tid, tag);   // (T > 4 only)
        if (T <= 8) router_rows<H, 8>(p, wg, G, tid, tag, red);
        else router_rows<H, kTMax>(p, wg, G, tid, tag, red);
    }
    if (tid == 0) stamp(p.stamps, wg, kStRouter);
    // One token (the ONE specialisation, launched for T = 1 without the timeout test hook):
    // its selected experts are the active experts, one slot per top-k position, so the work
    // partition is known before the ranking ends.  The helper wavefront ranks and
    // publishes each selection as soon as its round ends (f_rank); the compute wavefronts
    // quantise the token meanwhile (f_xq) and each starts streaming as soon as the
    // selections its units need are published.  No barrier and no metadata pass.
    bool ok = true;
    int U = 0;
    if constexpr (ONE) {
        U = K;
        if (wv == kWaves - 1) {
            if (p.inj_ids) {
                if (lane < K) {
                    sel_ids[lane] = p.inj_ids[lane];
                    sel_w[lane] = p.inj_w[lane];
                }
                if (lane == 0) lds_st(&f_rank, K);
            } else {
                const uint64_t* rows[1] = {p.logits};
                int* ids[1] = {sel_ids};
                uint64_t* stl = p.stamps ? p.stamps + wg * kStamps + kStLogits : nullptr;
                uint64_t* sts = p.stamps ? p.stamps + wg * kStamps + kStSelected : nullptr;
                ok = topk_bucket<1>(rows, E, K, lane, tag, status, limit, ids, p.policy, p.sel_bias, stl, sts,
                                    &f_rank);
            }
            if (ok) {   // the helper's own tables (token 0 at top-k position u of slot u)
                if (lane < K) {
                    const int e = sel_ids[lane];
                    if (e < 0 || e >= E) set_status(status, kDevBadIds);
                    act_e[lane] = e;
                    act_m[lane] = 1u;
                    act_j[lane * kTMax] = (uint8_t)lane;
                    if (wg == 0 && p.d_ids) p.d_ids[lane] = e;
                }
                lgkm_drain();
            } else {
                lds_st(&f_abort, 1);
            }
            if (lane == 0) stamp(p.stamps, wg, kStTopk);
        } else {
            quantise_input<H, kComputeWaves * 64>(p.x, 1, xq_s, xs_s, tid, wg == 0 ? p.d_xq : nullptr, p.d_xs);
            if (lane == 0) lds_add(&f_xq, 1);
            if (tid == 0) stamp(p.stamps, wg, kStQuant);
        }
    } else {
        // Input quantisation.  A small input (at most kLocalQuantChunks chunks per thread) is
        // quantised by every workgroup into its own LDS while the other router rows complete
        // (no exchange, and the work hides behind the logit wait).  A larger one is quantised
        // once, split over the workgroups (published before the router rows, above), and
        // fetched back: one round trip instead of G-fold replicated arithmetic.
        bool xq_ok = true;
        if (xq_exchange) {
            xq_ok = fetch_input<H>(p, T, xq_s, xs_s, tid, tag, status, limit);
        } else {
            quantise_input<H>(p.x, T, xq_s, xs_s, tid, wg == 0 ? p.d_xq : nullptr, p.d_xs);
        }
        if (tid == 0) stamp(p.stamps, wg, kStQuant);
        if (!xq_ok && lane == 0) s_fail = 1;   // read after the barrier that follows top-k

        // ---------------- stage 1: top-k (on the tagged logits), compact metadata ----------------
        if (p.fail_flag) {   // test hook: a wait that never completes, to exercise the timeout path
            if (tid == 0) {
                const uint64_t t0 = now();
                while (ld_co(status) == kDevOk && now() - t0 <= limit) __builtin_amdgcn_s_sleep(2);
                set_status(status, kDevTimeout);
                s_fail = 1;
            }
        } else if (p.inj_ids) {
            for (int i = tid; i < T * K; i += kThreads) {
                sel_ids[i] = p.inj_ids[i];
                sel_w[i] = p.inj_w[i];
            }
        } else {
            // two tokens per wavefront, interleaved (a lone last token runs on its own)
            for (int t0 = 2 * wv; t0 < T; t0 += 2 * kWaves) {
                const int t1 = min(t0 + 1, T - 1);
                const uint64_t* rows[2] = {p.logits + (size_t)t0 * E, p.logits + (size_t)t1 * E};
                int* ids[2] = {sel_ids + t0 * K, (t0 + 1 < T) ? sel_ids + t1 * K : nullptr};
                uint64_t* stl = (p.stamps && t0 == 0) ? p.stamps + wg * kStamps + kStLogits : nullptr;
                uint64_t* sts = (p.stamps && t0 == 0) ? p.stamps + wg * kStamps + kStSelected : nullptr;
                const bool good =
                    (t0 + 1 < T) ? topk_bucket<2>(rows, E, K, lane, tag, status, limit, ids, p.policy, p.sel_bias, stl, sts)
                                 : topk_bucket<1>(rows, E, K, lane, tag, status, limit, ids, p.policy, p.sel_bias, stl, sts);
                if (!good) {
                    if (lane == 0) s_fail = 1;
                    break;
                }
            }
        }
        __syncthreads();
        ok = s_fail == 0;
        if (ok) {
            if (tid == 0) stamp(p.stamps, wg, kStTopk);
            for (int i = tid; i < T * K; i += kThreads) {
                const int e = sel_ids[i];
                if (e >= 0 && e < E) atomicOr(&emask[e], 1u << (i / K));
                else set_status(status, kDevBadIds);
            }
            __syncthreads();
            if (tid == 0) stamp(p.stamps, wg, kStMask);
            if (wv == 0) {
                // compaction in expert order; emask[e] of an active expert becomes its slot
                // (one wavefront, so its own LDS writes are visible to its later reads)
                int base = 0;
                for (int e0 = 0; e0 < E; e0 += 64) {
                    const int e = e0 + lane;
                    const uint32_t msk = (e < E) ? emask[e] : 0u;
                    const uint64_t bal = __ballot(msk != 0u);
                    const int pre = __popcll(bal & ((1ull << lane) - 1ull));
                    if (msk) {
                        act_e[base + pre] = e;
                        act_m[base + pre] = msk;
                        emask[e] = (uint32_t)(base + pre);
                    }
                    base += __popcll(bal);
                }
                if (lane == 0) s_U = base;
                // pair table: top-k position of slot u in token t
                for (int i = lane; i < T * K; i += 64) {
                    const int e = sel_ids[i];
                    if (e >= 0 && e < E) act_j[emask[e] * kTMax + i / K] = (uint8_t)(i % K);
                }
            }
            if (wg == 0 && p.d_ids)
                for (int i = tid; i < T * K; i += kThreads) p.d_ids[i] = sel_ids[i];
            __syncthreads();
            U = uni(s_U);
            if (tid == 0) stamp(p.stamps, wg, kStMeta);
        }
    }

    // ---------------- work partition (identical in every wavefront) ----------------
    // Gate/up units are dealt round-robin over the workgroups (by default single units: the
    // j-th unit of workgroup wg is unit wg + G*j; the schedule may deal blocks of 2^up_lb
    // consecutive units instead).  Each expert's units are spread over many workgroups and every
    // workgroup works through the experts in slot order, so all workgroups stream the same
    // few experts at a time and the act rows complete expert by expert through the phase
    // (and with one token every workgroup starts on one of the first selections).  Down
    // units are split into contiguous ranges (one or two experts per workgroup, so each
    // workgroup requantises one or two act rows) over the first Gd workgroups (by default
    // the whole grid).
    const int n_up = U * UPE, n_dn = U * DNE;
    static_assert((uint64_t)kUMax * (H / 16) * kGridMax < (1ull << 32) &&
                      (uint64_t)kUMax * (I / 8) + ((uint64_t)kGridMax << kUpBlockLogMax) < (1ull << 31), "partition arithmetic");
    const int ulb = p.up_lb, Gd = p.dn_grid;
    const int nu = up_count(wg, G, n_up, ulb);                // gate/up units of this workgroup
    const int dlo = down_lo(wg, Gd, n_dn);
    const int dhi = down_lo(wg + 1, Gd, n_dn);
    const int nd = dhi - dlo;                                 // down units of this workgroup
    const int dn_u0 = nd > 0 ? dlo / DNE : 0;                 // first expert slot of the down range

    if (ok && wv < NC) {
        // ====================== compute wavefronts ======================
        // Work comes in tasks of two consecutive 128-deep blocks (256 deep) of one unit.
        // Within a phase the workgroup's tasks form one flat list dealt round-robin over
        // the compute wavefronts (wave w takes tasks w, w+NC, ...), so the waves stay
        // balanced whatever the tasks per unit.  A wave's share of one unit is a run of
        // tasks counted down on the hot path; at the end of the run the wave writes its
        // partial sums into the unit's hand-off slot.  Cursor state is wave-uniform
        // (scalar registers); the hot path advances pointers by constant strides and
        // branches only when a run ends.
        const int r16 = lane & 15;         // A row / B column (token) of this lane
        const int kq = lane >> 4;          // K quarter inside a 128-deep block
        const int rowc = min(r16, T - 1);  // B row read by this lane (dead columns have scale 0)
        constexpr int kTaskA = NC * 256;   // A bytes between a wave's consecutive tasks
        constexpr int kRunEnd = 1 << 30;   // countdown value once a cursor is exhausted
        // this wave's share of phase-relative unit r with NP tasks: first task kp0, count.
        // Whole units (NP < NC) go to wave r mod NC; otherwise the unit's task 0 goes to
        // wave (r*NP) mod NC and every wave has at least one task (NP >= NC).
        static_assert((NC & (NC - 1)) == 0, "wave count is a power of two");
        auto share = [&](int r, int NP, int& kp0) -> int {
            if (NP < NC) {
                kp0 = 0;
                return NP;
            }
            kp0 = (NP % NC == 0) ? wv : ((wv - r * NP) & (NC - 1));
            return (NP % NC == 0) ? NP / NC : (NP - 1 - kp0) / NC + 1;
        };
        // the first unit >= m of a phase (units are this workgroup's sequence numbers in the
        // phase) in which this wave has tasks
        auto own = [&](int m, int NP) -> int { return NP < NC ? m + ((wv - m) & (NC - 1)) : m; };
        // from (ph, m) on, the first unit in which this wave has tasks (ph = 2: none left);
        // closed form, no search; returned by value so the cursors stay in registers
        struct Pos { int ph, m, kp, cnt; };
        auto seek = [&](int ph, int m) -> Pos {
            if (ph == 0) {
                m = own(m, HP);
                if (m < nu) {
                    int kp;
                    const int cnt = share(m, HP, kp);
                    return Pos{0, m, kp, cnt};
                }
                m = 0;
            }
            if (ph <= 1) {
                m = own(m, IP);
                if (m < nd) {
                    int kp;
                    const int cnt = share(m, IP, kp);
                    return Pos{1, m, kp, cnt};
                }
            }
            return Pos{2, m, 0, 0};
        };
        // One-token path: before the first load of a unit of expert slot u, wait until the
        // selection of slot u is published (slots are top-k positions, ranked in order).  An
        // undetermined selection (-1) is reported by the helper; its address is clamped.
        auto ranked = [&](int u) MONOMOE_CURSOR_INLINE {
            if (lds_ld(&f_rank) <= u) {
                const uint64_t t0 = now();
                while (lds_ld(&f_rank) <= u) {
                    if (lds_ld(&f_abort) || now() - t0 > limit) {
                        set_status(status, kDevTimeout);
                        lds_st(&f_abort, 1);   // the waits that follow see the abort
                        break;
                    }
                    __builtin_amdgcn_s_sleep(1);
                }
            }
            compiler_fence();   // the selection is read after its counter
        };
        const Pos p0 = seek(0, 0);
        const int ph0 = p0.ph, m0 = p0.m, kp00 = p0.kp, cnt0 = p0.cnt;
        if (wv == 0 && lane == 0) stamp(p.stamps, wg, kStSeek);

        // ---- load cursor (RING tasks ahead of the compute cursor) ----
        int lph = ph0, lm = m0, lkp = kp00, lrem = cnt0;
        const uint8_t* lptr = p.w13;           // this lane's A bytes of the task
        const float* lsb = p.w13s;             // weight-scale array of the task's phase (uniform)
        uint32_t lso = 0;                      // this lane's scale index (two adjacent blocks)
        int lstep = 0, lsstep = 0;             // strides of the phase; 0 once exhausted (the last task reloads)
        auto lbase = [&]() MONOMOE_CURSOR_INLINE {   // per-lane addresses of task lkp of unit lm
            const int kb = 2 * lkp;
            if (lph == 0) {
                const int mu = up_unit(wg, G, lm, ulb);   // the unit
                const int u = mu / UPE, i0 = (mu - u * UPE) * 8;
                if constexpr (ONE) ranked(u);
                const int e = ONE ? min(max(uni(sel_ids[u]), 0), E - 1) : uni(act_e[u]);
                const int row = (r16 < 8) ? (i0 + r16) : (I + i0 + r16 - 8);
                lptr = p.w13 + ((size_t)e * 2 * I + row) * H + kb * 128 + kq * 16;
                const int rb = (lane < 32) ? (i0 >> 7) : ((I + i0) >> 7);
                lso = (uint32_t)((e * (2 * I / 128) + rb) * HB + kb);
                lsb = p.w13s;
                lstep = (HP < NC) ? 256 : kTaskA;
                lsstep = (HP < NC) ? 2 : NC * 2;
            } else {
                const int mu = dlo + lm;   // the unit
                const int u = mu / DNE, ht = mu - u * DNE;
                if constexpr (ONE) ranked(u);
                const int e = ONE ? min(max(uni(sel_ids[u]), 0), E - 1) : uni(act_e[u]);
                lptr = p.w2 + ((size_t)e * H + ht * 16 + r16) * I + kb * 128 + kq * 16;
                lso = (uint32_t)((e * HB + (ht >> 3)) * IB + kb);
                lsb = p.w2s;
                lstep = (IP < NC) ? 256 : kTaskA;
                lsstep = (IP < NC) ? 2 : NC * 2;
            }
        };
        auto lnext = [&]() MONOMOE_CURSOR_INLINE {   // once exhausted the cursor stays on its last task (reloads it)
            if (__builtin_expect(--lrem != 0, 1)) {
                lptr += lstep;
                lso += lsstep;
                return;
            }
            const Pos q = seek(lph, lm + 1);
            lph = q.ph;
            lm = q.m;
            lkp = q.kp;
            lrem = q.cnt;
            if (lph == 2) {
                lrem = kRunEnd;
                lstep = 0;
                lsstep = 0;
            } else {
                lbase();
            }
        };
        // weight-stream ring: slot s holds the A operands (two blocks) and the two weight
        // scales of one task.  Every ring step issues exactly five vector loads, so the
        // compiler's vmcnt bookkeeping stays exact and each use waits only for its slot.
        v4i ra[RING][4];
        float2 rws[RING];
        auto issue = [&](int s) {
            ra[s][0] = *reinterpret_cast<const v4i*>(lptr);
            ra[s][1] = *reinterpret_cast<const v4i*>(lptr + 64);
            ra[s][2] = *reinterpret_cast<const v4i*>(lptr + 128);
            ra[s][3] = *reinterpret_cast<const v4i*>(lptr + 192);
            rws[s] = *reinterpret_cast<const float2*>(lsb + lso);
        };

        // ---- compute cursor ----
        int cph = ph0, cm = m0, ckp = kp00, crem = cnt0;
        const uint8_t* bptr = xq_s;   // this lane's B operand (LDS) of the current task
        const float* sptr = xs_s;     // this lane's two activation scales (LDS; 0 for dead columns)
        int bstep = 0, sstep = 0;     // strides of the phase
        bool aborted = false;
        bool xq_ready = !ONE;
        auto cbase = [&]() -> bool {   // operand pointers (and readiness) for task ckp of unit cm
            const int kb = 2 * ckp;
            if (cph == 0) {
                if (!xq_ready) {   // one-token path: every compute wavefront's share of the input
                    if (!wait_lds(&f_xq, NC, &f_abort, limit)) return false;
                    xq_ready = true;
                }
                bptr = xq_s + rowc * XROW + kb * 128 + kq * 16;
                sptr = xs_s + r16 * HB + kb;
                bstep = (HP < NC) ? 256 : kTaskA;
                sstep = (HP < NC) ? 2 : NC * 2;
            } else {
                const int x = (dlo + cm) / DNE - dn_u0;   // this workgroup's x-th expert
                const int buf = (naq == 2) ? (x & 1) : 0;
                if (!wait_lds(&f_aq_seq[buf], x + 1, &f_abort, limit)) return false;
                const uint8_t* aq_s = lds_dyn + buf * aq_bytes;
                bptr = aq_s + rowc * AROW + kb * 128 + kq * 16;
                sptr = reinterpret_cast<const float*>(aq_s + T * AROW) + r16 * IB + kb;
                bstep = (IP < NC) ? 256 : kTaskA;
                sstep = (IP < NC) ? 2 : NC * 2;
            }
            return true;
        };
        bool stamped = false;
        auto handoff = [&](const v4f& acc) -> bool {   // partial sums of unit cm to the helper
            if constexpr (NCD == 1) {
                if (cph == 1) {
                    // A down unit computed by this wave alone: its epilogue (routing weight,
                    // tagged contribution) runs here instead of on the helper, and the wave's
                    // progress (its next unit) tells the helper when an activation buffer is free.
                    const int mu = dlo + cm, u = mu / DNE, ht = mu - u * DNE;
                    const uint32_t tmask = act_m[u];
                    const int c = lane & 15;
                    MONOMOE_PERTURB(4, cm);
                    if (c < T && ((tmask >> c) & 1u)) {
                        const int pi = c * K + act_j[u * kTMax + c];
                        const float w = sel_w[pi];
                        const uint64_t th = (uint64_t)tag << 32;
                        uint64_t* dst = p.contrib + (size_t)pi * H + ht * 16 + 4 * (lane >> 4);
#pragma unroll
                        for (int q = 0; q < 4; ++q) st_co(dst + q, th | __float_as_uint(acc[q] * w));
                    }
                    if (lane == 0) lds_st(&f_dn_prog[wv], cm + NC);   // (after this wave's buffer reads)
                    return true;
                }
            }
            const int useq = (cph == 0) ? cm : (nu + cm);
            const int slot = useq & smask;
            MONOMOE_PERTURB(1, useq);
            if (!wait_lds(&f_consumed, useq - smask, &f_abort, limit)) return false;
            part[(slot * NC + wv) * 64 + lane] = acc;
            if (lane == 0) lds_add(&f_cnt[slot], 1);
            if (!stamped) {
                stamped = true;
                if (wv == 0 && lane == 0) stamp(p.stamps, wg, kStFirstMfma);
            }
            return true;
        };

        if (ph0 != 2) {
            lbase();
            if (wv == 0 && lane == 0 && lptr != nullptr) stamp(p.stamps, wg, kStLbase);
#pragma clang loop unroll(full)
            for (int s = 0; s < RING; ++s) {   // prologue: fill the ring
                issue(s);
                lnext();
            }
            if (wv == 0 && lane == 0) stamp(p.stamps, wg, kStIssued);
            if (!cbase()) aborted = true;
            v4f acc = {0.f, 0.f, 0.f, 0.f};
            while (cph != 2 && !aborted) {
                // constant trip count (no early exit) so the ring stays in registers; the
                // loads are issued unconditionally (exact vmcnt bookkeeping), but once the
                // wave's work is done the remaining steps neither wait for nor use them
#pragma clang loop unroll(full)
                for (int s = 0; s < RING; ++s) {
                    const bool live = cph != 2;   // uniform
                    if (live) {
                        const v4i b0 = *reinterpret_cast<const v4i*>(bptr);
                        const v4i b1 = *reinterpret_cast<const v4i*>(bptr + 64);
                        const v4i b2 = *reinterpret_cast<const v4i*>(bptr + 128);
                        const v4i b3 = *reinterpret_cast<const v4i*>(bptr + 192);
                        const float2 as2 = *reinterpret_cast<const float2*>(sptr);
                        // gate/up: exact fp16 products (its output is requantised);
                        // down: the e4m3 MFMA
                        v4f blk0, blk1;
                        if (cph == 0) {
                            blk0 = block_mma(ra[s][0], ra[s][1], b0, b1);
                            blk1 = block_mma(ra[s][2], ra[s][3], b2, b3);
                        } else {
                            blk0 = block_mma_f8(ra[s][0], ra[s][1], b0, b1);
                            blk1 = block_mma_f8(ra[s][2], ra[s][3], b2, b3);
                        }
                        acc += blk0 * (rws[s].x * as2.x);
                        acc += blk1 * (rws[s].y * as2.y);
                        if (s == 0 && !stamped && wv == 0 && lane == 0 && acc[0] == acc[0] && p.stamps &&
                            p.stamps[wg * kStamps + kStFirstData] == 0)
                            stamp(p.stamps, wg, kStFirstData);
                    }
                    // refill this slot with the task RING ahead (unconditionally)
                    issue(s);
                    lnext();
                    if (!live) continue;
                    if (__builtin_expect(--crem != 0, 1)) {
                        bptr += bstep;
                        sptr += sstep;
                    } else {   // this wave's run of unit cm is done
                        if (!handoff(acc)) aborted = true;
                        acc = v4f{0.f, 0.f, 0.f, 0.f};
                        ++cm;
                        const int pph = cph;
                        const Pos q = seek(cph, cm);
                        cph = q.ph;
                        cm = q.m;
                        ckp = q.kp;
                        crem = q.cnt;
                        if (pph == 0 && cph != 0 && wv == 0 && lane == 0) stamp(p.stamps, wg, kStUpComputed);
                        if (cph == 2 || aborted) {
                            cph = 2;
                            crem = kRunEnd;
                        } else if (!cbase()) {
                            aborted = true;
                        }
                    }
                }
            }
            if (aborted) set_status(status, kDevTimeout);
            if (wv == 0 && lane == 0) stamp(p.stamps, wg, kStComputeDone);
            if (NCD == 1 && wv == 0 && lane == 0) stamp(p.stamps, wg, kStDownDone);
        }
        if (NCD == 1 && lane == 0) lds_st(&f_dn_prog[wv], 1 << 30);   // no unit left (also after an abort)
    } else if (ok) {
        // ====================== helper wavefront ======================
        bool fine = true;
        const uint64_t tag_hi = (uint64_t)tag << 32;
        // routing weights: needed only by the down epilogue, so they are computed here, off
        // the path from routing to the first weight loads (injected weights are kept)
        if (!p.inj_ids) routing_weights<kTMax * kKMax / 64>(p.logits, sel_ids, sel_w, T, E, K, p.renorm, p.policy, p.route_scale, lane);
        if (wg == 0 && p.d_w)
            for (int i = lane; i < T * K; i += 64) p.d_w[i] = sel_w[i];

        // --- gate/up epilogues: SiLU(gate)*up, stored as tagged words ---
        for (int j = 0; j < nu; ++j) {
            const int m = up_unit(wg, G, j, ulb), slot = j & smask;
            if (!wait_lds(&f_cnt[slot], NCU, &f_abort, limit)) { fine = false; break; }
            const int u = m / UPE, i0 = (m - u * UPE) * 8;
            const uint32_t tmask = act_m[u];
            v4f gs = {0.f, 0.f, 0.f, 0.f}, us = {0.f, 0.f, 0.f, 0.f};
            if (lane < 32) {
#pragma unroll
                for (int b = 0; b < NCU; ++b) {
                    const int v = (HP >= NC) ? b : (j % NC);   // b-th contributor
                    gs += part[(slot * NC + v) * 64 + lane];
                    us += part[(slot * NC + v) * 64 + lane + 32];
                }
            }
            lds_st(&f_cnt[slot], 0);
            lds_st(&f_consumed, j + 1);
            MONOMOE_PERTURB(2, j);
            const int c = lane & 15;
            if (lane < 32 && c < T && ((tmask >> c) & 1u)) {
                v4f a;
#pragma unroll
                for (int q = 0; q < 4; ++q) a[q] = gs[q] / (1.0f + expf(-gs[q])) * us[q];
                const size_t pi = (size_t)c * K + act_j[u * kTMax + c];
                uint64_t* dst = p.act + pi * I + i0 + 4 * (lane >> 4);
#pragma unroll
                for (int q = 0; q < 4; ++q) st_co(dst + q, tag_hi | __float_as_uint(a[q]));
                if (p.d_act) *reinterpret_cast<v4f*>(p.d_act + pi * I + i0 + 4 * (lane >> 4)) = a;
            }
        }
        if (lane == 0) stamp(p.stamps, wg, kStUpDone);

        // --- down: requantise the next expert's activation into LDS, then the epilogues ---
        const int nx = nd > 0 ? (dhi - 1) / DNE - dn_u0 + 1 : 0;
        int prepared = 0;
        // prepare(x): poll the tagged SiLU activations of every routed token of expert slot
        // dn_u0 + x and requantise them per 128-group into LDS buffer x % naq (16 lanes per
        // group, 8 values each).  Non-blocking mode gives up at the first group that is not
        // complete yet (the buffer is not in use, and is rewritten on the next attempt).
        auto prepare = [&](int x, bool block) -> bool {
            const int u = dn_u0 + x;
            const int buf = (naq == 2) ? (x & 1) : 0;
            uint8_t* aq_s = lds_dyn + buf * aq_bytes;
            float* as_s = reinterpret_cast<float*>(aq_s + T * AROW);
            uint32_t tm = (uint32_t)uni((int)act_m[u]);
            const int cnt = __popc(tm);
            for (int q = 0; q < cnt; ++q) {
                const int t = __ffs(tm) - 1;
                tm &= tm - 1u;
                if (lane == 0) {
                    h_t[q] = t;
                    h_pi[q] = t * K + act_j[u * kTMax + t];
                }
            }
            for (int i = lane; i < kTMax * IB; i += 64) as_s[i] = 0.0f;   // unrouted tokens: scale 0
            lgkm_drain();
            const __amdgpu_buffer_rsrc_t ra = buf_rsrc(p.act);
            const int ngr = cnt * IB;
            const uint64_t t0 = now();
            // kPB batches of four groups are polled per round trip (an expert with several
            // routed tokens has many groups; one round trip per batch would serialise them)
            constexpr int kPB = 2;
            for (int g00 = 0; g00 < ngr; g00 += 4 * kPB) {
                uint32_t off[kPB];
#pragma unroll
                for (int b = 0; b < kPB; ++b) {
                    const int gi = min(g00 + 4 * b + (lane >> 4), ngr - 1);
                    const int q = gi / IB, g = gi - q * IB;
                    off[b] = (uint32_t)((h_pi[q] * I + g * 128 + 8 * (lane & 15)) * 8);
                }
                v4i d[kPB][4];
                while (true) {
#pragma unroll
                    for (int b = 0; b < kPB; ++b)
#pragma unroll
                        for (int i = 0; i < 4; ++i) d[b][i] = ld_co16(ra, off[b] + 16u * i);
                    bool fresh = true;
#pragma unroll
                    for (int b = 0; b < kPB; ++b)
#pragma unroll
                        for (int i = 0; i < 4; ++i)
                            fresh = fresh && (uint32_t)d[b][i][1] == tag && (uint32_t)d[b][i][3] == tag;
                    if (__ballot(!fresh) == 0) break;
                    if (!block) return false;
                    if (ld_co(status) != kDevOk) return false;
                    if (now() - t0 > limit) {
                        set_status(status, kDevTimeout);
                        return false;
                    }
                    __builtin_amdgcn_s_sleep(1);
                }
#pragma unroll
                for (int b = 0; b < kPB; ++b) {
                    const int g0 = g00 + 4 * b;
                    if (g0 >= ngr) break;   // uniform
                    const int gi = min(g0 + (lane >> 4), ngr - 1);
                    const int q = gi / IB, g = gi - q * IB;
                    float f[8];
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        f[2 * i] = __int_as_float(d[b][i][0]);
                        f[2 * i + 1] = __int_as_float(d[b][i][2]);
                    }
                    float a = 0.0f;
#pragma unroll
                    for (int i = 0; i < 8; ++i) a = fmaxf(a, fabsf(f[i]));
                    const float amax = row16_max(a);
                    float sc = e4m3_scale(amax);
                    uint32_t c0 = 0u, c1 = 0u;
                    if (amax == 0.0f || sc == 0.0f) {
                        sc = 0.0f;
                    } else {
                        const double r = 1.0 / (double)sc;
                        c0 = e4m3x2(quot_rn(f[0], r), quot_rn(f[1], r)) | (e4m3x2(quot_rn(f[2], r), quot_rn(f[3], r)) << 16);
                        c1 = e4m3x2(quot_rn(f[4], r), quot_rn(f[5], r)) | (e4m3x2(quot_rn(f[6], r), quot_rn(f[7], r)) << 16);
                    }
                    if (g0 + (lane >> 4) < ngr) {
                        const int t = h_t[q];
                        *reinterpret_cast<uint2*>(aq_s + t * AROW + g * 128 + 8 * (lane & 15)) = make_uint2(c0, c1);
                        if ((lane & 15) == 0) as_s[t * IB + g] = sc;
                        if (p.d_aq) {
                            *reinterpret_cast<uint2*>(p.d_aq + (size_t)h_pi[q] * I + g * 128 + 8 * (lane & 15)) =
                                make_uint2(c0, c1);
                            if ((lane & 15) == 0) p.d_as[h_pi[q] * IB + g] = sc;
                        }
                    }
                }
            }
            lds_st(&f_aq_seq[buf], x + 1);
            return true;
        };
        if constexpr (NCD == 1) {
            // Down units are computed and stored by the compute wavefronts (direct epilogues):
            // the helper only requantises each expert of the range into its buffer, once the
            // buffer's previous expert (x - naq) has no unit left to compute.
            for (int x = 0; x < nx && fine; ++x) {
                if (x >= naq) {
                    const int J = max(0, (dn_u0 + x - naq + 1) * DNE - dlo);   // first unit of expert x - naq + 1
                    for (int w = 0; w < NC && fine; ++w)
                        if (!wait_lds(&f_dn_prog[w], J, &f_abort, limit)) fine = false;
                    if (!fine) break;
                }
                MONOMOE_PERTURB(3, x);
                if (!prepare(x, true)) { fine = false; break; }
                if (x == 0 && lane == 0) stamp(p.stamps, wg, kStFirstAq);
            }
        }
        for (int j = 0; NCD != 1 && j < nd && fine; ++j) {
            const int m = dlo + j, u = m / DNE, ht = m - u * DNE, x = u - dn_u0;
            const int useq = nu + j, slot = useq & smask;
            while (prepared <= x) {
                MONOMOE_PERTURB(3, prepared);
                if (!prepare(prepared, true)) { fine = false; break; }
                if (prepared == 0 && lane == 0) stamp(p.stamps, wg, kStFirstAq);
                prepared += 1;
            }
            if (!fine) break;
            if (naq == 2 && prepared == x + 1 && prepared < nx) {
                if (prepare(prepared, false)) prepared += 1;
            }
            if (!wait_lds(&f_cnt[slot], NCD, &f_abort, limit)) { fine = false; break; }
            v4f y = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int b = 0; b < NCD; ++b) y += part[(slot * NC + ((IP >= NC) ? b : (j % NC))) * 64 + lane];
            lds_st(&f_cnt[slot], 0);
            lds_st(&f_consumed, useq + 1);
            MONOMOE_PERTURB(4, j);
            const uint32_t tmask = act_m[u];
            const int c = lane & 15;
            if (c < T && ((tmask >> c) & 1u)) {   // this token's weighted contribution, tagged
                const int pi = c * K + act_j[u * kTMax + c];
                const float w = sel_w[pi];
                uint64_t* dst = p.contrib + (size_t)pi * H + ht * 16 + 4 * (lane >> 4);
#pragma unroll
                for (int q = 0; q < 4; ++q) st_co(dst + q, tag_hi | __float_as_uint(y[q] * w));
            }
        }
        if (NCD != 1 && lane == 0) stamp(p.stamps, wg, kStDownDone);
        if (!fine) {
            set_status(status, kDevTimeout);
            lds_st(&f_abort, 1);
        }
    }

    // ---------------- final reduction: the output chunks this workgroup owns ----------------
    // The output is dealt in chunks of 64 (16 columns of one tile x 4 tokens): chunk
    // r = c * (H/16) + ht (tile ht, tokens 4c .. 4c+3) goes to workgroup r mod G, one
    // wavefront per chunk.  Every token's k tagged contributions are polled and summed in
    // top-k order (a fixed order, so the output does not depend on timing), then rounded to
    // bf16.
    __syncthreads();
    if (ok && ld_co(status) == kDevOk) {
        const int nchunk = (H / 16) * ((T + 3) / 4);
        for (int r = wg + G * wv; r < nchunk; r += G * kWaves) {
            const int c = r / (H / 16), ht = r - c * (H / 16);
            MONOMOE_PERTURB(5, r);
            if (!reduce_chunk<H>(p, ht, 64 * c, T, K, tag, lane, status, limit)) break;
        }
    }
    if (tid == 0) stamp(p.stamps, wg, kStReduced);

    // ---------------- exit: this workgroup's launch count advances ----------------
    __syncthreads();
    if (tid == 0) {
        stamp(p.stamps, wg, kStExit);
        st_co(ctl + kCtlEpoch + wg, tag);
    }
}

template <int H, int I, int RING, bool ONE>
static void launch_fused(const KParams& p, int grid, size_t lds, hipStream_t stream) {
    hipLaunchKernelGGL((monomoe_fused<H, I, RING, ONE>), dim3(grid), dim3(kThreads), lds, stream, p);
}

}  // namespace monomoe
