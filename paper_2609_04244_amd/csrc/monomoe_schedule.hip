// Host-side model check of the single-tile kernel's hand-off protocol (monomoe_schedule_check).
//
// The kernel's readiness-based hand-offs (Sec. 3.2) are safe only if every wait is eventually
// satisfied and no producer overwrites data before its consumer has read it.  This file
// replays, for one routing, every wavefront's synchronisation events in the order the kernel
// issues them, with the kernel's own work-partition arithmetic (monomoe_partition.h), and
// executes them under a scheduler that interleaves the wavefronts in a seeded pseudo-random
// order with a bounded number of resident workgroups.  Modelled per workgroup: the router-row
// barriers, the input exchange, the selection (and, with one token, the progressive
// publication of each top-k position and the compute wavefronts' quantisation counter), the
// barriers of the metadata pass, the partial-sum hand-off slot ring (f_cnt / f_consumed), the
// requantised-activation buffers (f_aq_seq, one or two buffers, blocking and non-blocking
// preparation), the activation and contribution words, and the output reduction.  Data
// values are not modelled; the checks are progress (no deadlock) and the safety of every LDS
// reuse.  Waits are modelled as the kernel writes them; where a wavefront polls a subset of
// a set of words (input groups), the model waits for the whole set, which can only add
// blocking, so a complete run of the model implies a complete run of the kernel's order.
#include <stdint.h>
#include <stdlib.h>

#include <algorithm>
#include <vector>

#include "monomoe.h"
#include "monomoe_internal.h"
#include "monomoe_partition.h"

namespace monomoe {
namespace {

enum Ev : int8_t {
    kEvBarrier,         // arrive at the workgroup's next barrier, wait for all its wavefronts
    kEvPublishRow,      // a router row's logits (all tokens) stored
    kEvWaitRows,        // all router rows stored (a token's selection needs every logit)
    kEvPublishGroups,   // this wavefront's share of the exchanged input groups stored
    kEvWaitGroups,      // every share stored (the workgroup's copy of the quantised input)
    kEvRank,            // one token: top-k position a - 1 published (f_rank = a)
    kEvQuantDone,       // one token: this compute wavefront's quantisation share done (f_xq += 1)
    kEvWaitRanked,      // one token: load cursor entering a unit of expert slot a (f_rank > a)
    kEvWaitXq,          // one token: first gate/up unit (f_xq == compute wavefronts)
    kEvWaitAq,          // down unit of the workgroup's a-th expert: its buffer prepared
    kEvHandoff,         // partial sums of hand-off sequence number a (b: down expert or -1)
    kEvConsume,         // helper: sums of sequence number a (b: contributor count, c: contributor)
    kEvPublishAct,      // helper: activation words of gate/up unit a
    kEvPrepareUpTo,     // helper: blocking preparation of experts up to a
    kEvPrefetch,        // helper: non-blocking preparation of expert a + 1 (two buffers)
    kEvPublishContrib,  // helper: contribution words of down unit a
    kEvWaitContrib,     // reduction of output chunk a
    kEvDirect,          // down unit a (relative) computed by one wavefront alone: its contribution
                        // stored by that wavefront (b: down expert, c: its slot), progress a + NC
    kEvProgressEnd,     // compute wavefront: no down unit left (progress = infinity)
    kEvWaitProgress,    // helper: every compute wavefront's progress >= a
    kEvEnd,
};

enum : int {   // violation kinds (monomoe_schedule_report_t.first_violation)
    kVioSlotOverwrite = 1,   // a hand-off slot rewritten before the helper consumed it
    kVioSlotStale = 2,       // the helper consumed a slot that does not hold the expected sums
    kVioBufferRead = 3,      // a compute wavefront read an activation buffer holding another expert
    kVioBufferOverwrite = 4, // an activation buffer rewritten while a compute wavefront reads it
    kVioDuplicate = 5,       // a gate/up or down unit published twice (partition overlap)
};

struct Step {
    Ev ev;
    int a, b, c;
};

struct Wave {
    std::vector<Step> prog;
    size_t pc = 0;
    bool arrived = false;   // at the current barrier
    int reading = -1;       // compute wavefront: down expert whose buffer it reads
    int prepared = 0;       // helper: experts prepared
};

struct Group {
    int wg;
    int nu = 0, dlo = 0, nd = 0, nx = 0;   // gate/up units; the contiguous down range, its slots
    std::vector<int> barrier;     // arrivals per barrier index
    int f_rank = 0, f_xq = 0, f_consumed = 0;
    int f_aq_seq[2] = {0, 0};
    int f_dn_prog[kComputeWaves] = {0, 1, 2, 3};   // direct down epilogues: next unfinished unit per wave
    int content[2] = {-1, -1};    // expert slot held by each activation buffer (-2: partly written)
    std::vector<int> f_cnt;       // per slot
    std::vector<int> part;        // [slot][wave]: sequence number last written (-1: none)
    Wave w[kWaves];
    int started = 0, ended = 0;
};

struct Model {
    // shape and schedule
    int T, H, E, I, K, G, nslots, naq, one, ring;
    int ulb, Gd;                  // work partition: gate/up deal block 2^ulb, down workgroups
    int U, UPE, DNE, HP, IP, NCU, NCD;
    uint32_t mutate;
    bool exchange;
    // routing: slot of each (token, top-k position) pair; experts of each slot
    std::vector<int> pair_slot;
    // global facts
    int rows_done = 0, shares_done = 0;
    std::vector<uint8_t> act;       // gate/up unit published
    std::vector<int> act_slot;      // units published per expert slot
    std::vector<uint8_t> contrib;   // down unit published
    std::vector<Group> g;
    int64_t events = 0;
    int violations = 0, first_violation = 0;

    void violate(int kind) {
        if (violations++ == 0) first_violation = kind;
    }
};

constexpr int NC = kComputeWaves;

// wavefront wv's first task and task count in phase-relative unit r with NP tasks (the
// kernel's round-robin deal of tasks over the compute wavefronts)
int share(int wv, int r, int NP, int& kp0) {
    if (NP < NC) {
        kp0 = 0;
        return ((r & (NC - 1)) == wv) ? NP : 0;
    }
    kp0 = (NP % NC == 0) ? wv : ((wv - r * NP) & (NC - 1));
    return (NP % NC == 0) ? NP / NC : (NP - 1 - kp0) / NC + 1;
}

void build_compute(Model& M, Group& gr, int wv) {
    std::vector<Step>& P = gr.w[wv].prog;
    // the wavefront's tasks in order: (phase, phase-relative unit)
    struct Task { int ph, m; };
    std::vector<Task> tasks;
    for (int m = 0; m < gr.nu; ++m) {
        int kp;
        const int c = share(wv, m, M.HP, kp);
        for (int i = 0; i < c; ++i) tasks.push_back({0, m});
    }
    for (int m = 0; m < gr.nd; ++m) {
        int kp;
        const int c = share(wv, m, M.IP, kp);
        for (int i = 0; i < c; ++i) tasks.push_back({1, m});
    }
    auto slot_of = [&](const Task& t) {   // expert slot of a task's unit
        return t.ph == 0 ? up_unit(gr.wg, M.G, t.m, M.ulb) / M.UPE : (gr.dlo + t.m) / M.DNE;
    };
    auto new_unit = [&](size_t i) { return i == 0 || tasks[i].ph != tasks[i - 1].ph || tasks[i].m != tasks[i - 1].m; };
    auto lbase = [&](size_t i) {   // load cursor entering task i
        if (M.one && i < tasks.size() && new_unit(i)) P.push_back({kEvWaitRanked, slot_of(tasks[i]), 0, 0});
    };
    bool xq_ready = !M.one;
    auto cbase = [&](size_t i) {   // compute cursor entering the unit of task i
        const Task& t = tasks[i];
        if (t.ph == 0) {
            if (!xq_ready) {
                P.push_back({kEvWaitXq, 0, 0, 0});
                xq_ready = true;
            }
        } else {
            P.push_back({kEvWaitAq, (gr.dlo + t.m) / M.DNE - gr.dlo / M.DNE, 0, (gr.dlo + t.m) / M.DNE});
        }
    };
    if (tasks.empty()) {
        if (M.NCD == 1) P.push_back({kEvProgressEnd, 0, 0, 0});
        return;
    }
    const int ring = M.ring;   // the load cursor runs this many tasks ahead of the compute cursor
    lbase(0);
    for (int s = 0; s < ring; ++s) lbase((size_t)s + 1);
    cbase(0);
    for (size_t i = 0; i < tasks.size(); ++i) {
        lbase(i + ring + 1);
        const bool last = i + 1 == tasks.size() || new_unit(i + 1);
        if (last) {
            const Task& t = tasks[i];
            const int useq = t.ph == 0 ? t.m : gr.nu + t.m;
            const int u = t.ph == 0 ? -1 : (gr.dlo + t.m) / M.DNE;
            const int x = t.ph == 0 ? -1 : u - gr.dlo / M.DNE;
            if (t.ph == 1 && M.NCD == 1) P.push_back({kEvDirect, t.m, x, u});
            else P.push_back({kEvHandoff, useq, x, u});
            if (i + 1 < tasks.size()) cbase(i + 1);
        }
    }
    if (M.NCD == 1) P.push_back({kEvProgressEnd, 0, 0, 0});
}

void build_helper(Model& M, Group& gr) {
    std::vector<Step>& P = gr.w[kWaves - 1].prog;
    for (int j = 0; j < gr.nu; ++j) {
        const int v = M.HP >= NC ? -1 : (j % NC);
        P.push_back({kEvConsume, j, M.NCU, v});
        P.push_back({kEvPublishAct, up_unit(gr.wg, M.G, j, M.ulb), 0, 0});
    }
    if (M.NCD == 1) {   // direct down epilogues: the helper only prepares each expert's buffer
        for (int x = 0; x < gr.nx; ++x) {
            // the buffer's previous expert (x - naq) has no unit left; the one-buffer mutation
            // drops this wait
            if (x >= M.naq && !(M.mutate & MONOMOE_SCHEDULE_MUTATE_PREFETCH_ONE_BUFFER))
                P.push_back({kEvWaitProgress, std::max(0, (gr.dlo / M.DNE + x - M.naq + 1) * M.DNE - gr.dlo), 0, 0});
            P.push_back({kEvPrepareUpTo, x, 0, 0});
        }
        return;
    }
    for (int j = 0; j < gr.nd; ++j) {
        const int x = (gr.dlo + j) / M.DNE - gr.dlo / M.DNE;
        P.push_back({kEvPrepareUpTo, x, 0, 0});
        if (M.naq == 2 || (M.mutate & MONOMOE_SCHEDULE_MUTATE_PREFETCH_ONE_BUFFER)) P.push_back({kEvPrefetch, x, 0, 0});
        const int v = M.IP >= NC ? -1 : (j % NC);
        P.push_back({kEvConsume, gr.nu + j, M.NCD, v});
        P.push_back({kEvPublishContrib, gr.dlo + j, 0, 0});
    }
}

void build(Model& M) {
    const int n_up = M.U * M.UPE, n_dn = M.U * M.DNE;
    M.act.assign(n_up, 0);
    M.act_slot.assign(M.U, 0);
    M.contrib.assign(n_dn, 0);
    M.g.resize(M.G);
    const int nchunk = (M.H / 16) * ((M.T + 3) / 4);
    for (int wg = 0; wg < M.G; ++wg) {
        Group& gr = M.g[wg];
        gr.wg = wg;
        gr.nu = up_count(wg, M.G, n_up, M.ulb);
        gr.dlo = down_lo(wg, M.Gd, n_dn);
        gr.nd = down_lo(wg + 1, M.Gd, n_dn) - gr.dlo;
        gr.nx = gr.nd > 0 ? (gr.dlo + gr.nd - 1) / M.DNE - gr.dlo / M.DNE + 1 : 0;
        gr.f_cnt.assign(M.nslots, 0);
        gr.part.assign((size_t)M.nslots * NC, -1);
        int nbar = 0;
        for (int wv = 0; wv < kWaves; ++wv) {
            std::vector<Step>& P = gr.w[wv].prog;
            int b = 0;
            P.push_back({kEvBarrier, b++, 0, 0});   // flags initialised
            if (M.exchange) P.push_back({kEvPublishGroups, 0, 0, 0});   // the input share, first
            // stage 0: router rows e = wg, wg + G, ... (two workgroup barriers each; the
            // first wavefront's lanes store the row)
            for (int e = wg; e < M.E; e += M.G) {
                P.push_back({kEvBarrier, b++, 0, 0});
                if (wv == 0) P.push_back({kEvPublishRow, e, 0, 0});
                P.push_back({kEvBarrier, b++, 0, 0});
            }
            if (M.one) {
                if (wv == kWaves - 1) {
                    P.push_back({kEvWaitRows, 0, 0, 0});
                    for (int u = 1; u <= M.K; ++u) P.push_back({kEvRank, u, 0, 0});
                } else {
                    P.push_back({kEvQuantDone, 0, 0, 0});
                }
            } else {
                if (M.exchange) P.push_back({kEvWaitGroups, 0, 0, 0});
                if (2 * wv < M.T) P.push_back({kEvWaitRows, 0, 0, 0});   // this wavefront's tokens
                for (int i = 0; i < 3; ++i) P.push_back({kEvBarrier, b++, 0, 0});   // top-k, masks, metadata
            }
            if (wv < NC) build_compute(M, gr, wv);
            else build_helper(M, gr);
            P.push_back({kEvBarrier, b++, 0, 0});   // before the output reduction
            for (int r = wg + M.G * wv; r < nchunk; r += M.G * kWaves) P.push_back({kEvWaitContrib, r, 0, 0});
            P.push_back({kEvBarrier, b++, 0, 0});   // before the exit
            P.push_back({kEvEnd, 0, 0, 0});
            nbar = b;
        }
        gr.barrier.assign(nbar, 0);
    }
}


// Try to execute wavefront (gr, wv)'s next step; false when it is blocked (or ended).
bool step(Model& M, Group& gr, int wv) {
    Wave& W = gr.w[wv];
    const Step& s = W.prog[W.pc];
    const int smask = M.nslots - 1;
    auto buf = [&](int x) { return M.naq == 2 ? (x & 1) : 0; };
    // requantisation of expert x into its buffer: the writes begin with the first poll (group
    // by group as they complete, blocking or not), so the buffer must be free at every attempt;
    // an attempt that stops early leaves it partly written
    auto prepare = [&](int x) -> bool {
        const int b = buf(x), u = gr.dlo / M.DNE + x;
        for (int v = 0; v < NC; ++v)
            if (gr.w[v].reading >= 0 && gr.w[v].reading != x && buf(gr.w[v].reading) == b) M.violate(kVioBufferOverwrite);
        if (M.act_slot[u] < M.UPE) {   // an activation group of the expert is not complete
            gr.content[b] = -2;
            return false;
        }
        gr.content[b] = u;
        gr.f_aq_seq[b] = x + 1;
        return true;
    };
    switch (s.ev) {
        case kEvEnd:
            return false;
        case kEvBarrier:
            if (!W.arrived) {
                W.arrived = true;
                gr.barrier[s.a] += 1;
            }
            if (gr.barrier[s.a] < kWaves) return false;
            W.arrived = false;
            break;
        case kEvPublishRow:
            M.rows_done += 1;
            break;
        case kEvWaitRows:
            if (M.rows_done < M.E) return false;
            break;
        case kEvPublishGroups:
            M.shares_done += 1;
            break;
        case kEvWaitGroups:
            if (M.shares_done < M.G * kWaves) return false;
            break;
        case kEvRank:
            gr.f_rank = s.a;
            break;
        case kEvQuantDone:
            gr.f_xq += 1;
            break;
        case kEvWaitRanked:
            if (gr.f_rank <= s.a) return false;
            break;
        case kEvWaitXq:
            if (gr.f_xq < NC) return false;
            break;
        case kEvWaitAq: {
            const int b = buf(s.a);
            if (!(M.mutate & MONOMOE_SCHEDULE_MUTATE_NO_ACT_WAIT) && gr.f_aq_seq[b] < s.a + 1) return false;
            if (gr.content[b] != s.c) M.violate(kVioBufferRead);
            W.reading = s.a;
            break;
        }
        case kEvHandoff: {
            const int slot = s.a & smask;
            if (!(M.mutate & MONOMOE_SCHEDULE_MUTATE_NO_SLOT_WAIT) && gr.f_consumed < s.a - smask) return false;
            if (s.b >= 0 && gr.content[buf(s.b)] != s.c) M.violate(kVioBufferOverwrite);
            const int prev = gr.part[slot * NC + wv];
            if (prev >= 0 && gr.f_consumed <= prev) M.violate(kVioSlotOverwrite);
            gr.part[slot * NC + wv] = s.a;
            gr.f_cnt[slot] += 1;
            W.reading = -1;
            break;
        }
        case kEvConsume: {
            const int slot = s.a & smask;
            if (gr.f_cnt[slot] < s.b) return false;
            for (int v = 0; v < NC; ++v)
                if ((s.c < 0 || s.c == v) && gr.part[slot * NC + v] != s.a) M.violate(kVioSlotStale);
            gr.f_cnt[slot] = 0;
            gr.f_consumed = s.a + 1;
            break;
        }
        case kEvPublishAct:
            if (M.act[s.a]) M.violate(kVioDuplicate);
            M.act[s.a] = 1;
            M.act_slot[s.a / M.UPE] += 1;
            break;
        case kEvPrepareUpTo:
            if (W.prepared <= s.a) {
                if (!prepare(W.prepared)) return false;
                W.prepared += 1;
                if (W.prepared <= s.a) return true;   // more to prepare: same step again
            }
            break;
        case kEvPrefetch:
            // the next expert's buffer (two buffers; the mutation also with one), when its
            // activations are complete (non-blocking)
            if (W.prepared == s.a + 1 && W.prepared < gr.nx) {
                if (prepare(W.prepared)) W.prepared += 1;
            }
            break;
        case kEvPublishContrib:
            if (M.contrib[s.a]) M.violate(kVioDuplicate);
            M.contrib[s.a] = 1;
            break;
        case kEvDirect:
            if (gr.content[buf(s.b)] != s.c) M.violate(kVioBufferOverwrite);
            if (M.contrib[gr.dlo + s.a]) M.violate(kVioDuplicate);
            M.contrib[gr.dlo + s.a] = 1;
            W.reading = -1;
            gr.f_dn_prog[wv] = s.a + NC;
            break;
        case kEvProgressEnd:
            gr.f_dn_prog[wv] = 1 << 30;
            break;
        case kEvWaitProgress:
            for (int v = 0; v < NC; ++v)
                if (gr.f_dn_prog[v] < s.a) return false;
            break;
        case kEvWaitContrib: {
            const int ht = s.a % (M.H / 16), c = s.a / (M.H / 16);
            for (int t = 4 * c; t < std::min(4 * c + 4, M.T); ++t)
                for (int j = 0; j < M.K; ++j)
                    if (!M.contrib[M.pair_slot[t * M.K + j] * M.DNE + ht]) return false;
            break;
        }
    }
    W.pc += 1;
    M.events += 1;
    return true;
}

uint32_t next_rand(uint64_t& st) {   // xorshift64*
    st ^= st >> 12;
    st ^= st << 25;
    st ^= st >> 27;
    return (uint32_t)((st * 0x2545F4914F6CDD1Dull) >> 32);
}

}  // namespace
}  // namespace monomoe

using namespace monomoe;

extern "C" int monomoe_schedule_check(const monomoe_shape_t* shape, int topk, const int32_t* topk_ids,
                                      int one_token, int grid, int ring, int up_block, int down_grid,
                                      int handoff_slots, int act_buffers, int resident, uint32_t seed,
                                      uint32_t mutate,
                                      monomoe_schedule_report_t* out) {
    if (!shape || !topk_ids || !out) return MONOMOE_ERR_INVALID;
    const int T = shape->T, H = shape->H, E = shape->E, I = shape->I;
    if (T < 1 || H < 256 || I < 256 || H % 256 || I % 256 || E < 1 || E > kEMax || topk < 1 || topk > kKMax ||
        topk > E || grid < 1 || grid > kGridMax || resident < 1 || (one_token != 0 && one_token != 1) ||
        (ring != kRings[0] && ring != kRings[1]) || down_grid < 0 || down_grid > grid ||
        (up_block != 0 && up_block != 1 && up_block != 2 && up_block != 4 && up_block != 8) ||
        handoff_slots < 1 || (handoff_slots & (handoff_slots - 1)) || handoff_slots > kSlotsMax ||
        (act_buffers != 1 && act_buffers != 2) || (mutate & ~7u))
        return MONOMOE_ERR_INVALID;
    if (T > kTMax || (one_token && T != 1)) return MONOMOE_ERR_UNSUPPORTED;
    Model M;
    M.T = T, M.H = H, M.E = E, M.I = I, M.K = topk, M.G = grid, M.nslots = handoff_slots, M.naq = act_buffers;
    M.one = one_token, M.ring = ring, M.mutate = mutate;
    M.ulb = up_block >= 8 ? 3 : up_block >= 4 ? 2 : up_block >= 2 ? 1 : 0;
    M.Gd = down_grid == 0 ? grid : down_grid;
    M.UPE = I / 8, M.DNE = H / 16, M.HP = H / 256, M.IP = I / 256;
    M.NCU = M.HP < NC ? 1 : NC, M.NCD = M.IP < NC ? 1 : NC;
    M.exchange = !one_token && T * (H / 8) > kLocalQuantChunks * kThreads;
    // expert slots: with one token the top-k positions; otherwise the active experts in
    // expert order
    M.pair_slot.assign((size_t)T * topk, 0);
    std::vector<int> slot_of(E, -1);
    for (int t = 0; t < T; ++t)
        for (int j = 0; j < topk; ++j) {
            const int e = topk_ids[t * topk + j];
            if (e < 0 || e >= E) return MONOMOE_ERR_INVALID;
            for (int i = 0; i < j; ++i)
                if (topk_ids[t * topk + i] == e) return MONOMOE_ERR_INVALID;
            slot_of[e] = 0;
        }
    if (one_token) {
        M.U = topk;
        for (int j = 0; j < topk; ++j) M.pair_slot[j] = j;
    } else {
        int U = 0;
        for (int e = 0; e < E; ++e)
            if (slot_of[e] == 0) slot_of[e] = U++;
        M.U = U;
        for (int i = 0; i < T * topk; ++i) M.pair_slot[i] = slot_of[topk_ids[i]];
    }
    build(M);

    // Scheduler: workgroups start in index order, at most `resident` at a time, a new one
    // when one ends; each pass visits the running wavefronts in a pseudo-random order
    // (seed 0: in order) and runs each for 1..8 steps (seed 0: one) or until it blocks.  A
    // pass without progress while work remains is a deadlock.
    uint64_t st = seed ? 0x9E3779B97F4A7C15ull ^ ((uint64_t)seed * 0xD1B54A32D192ED03ull) : 1ull;
    int next_wg = 0, running = 0, finished = 0;
    std::vector<int> order;
    int blocked_wg = -1, blocked_wave = -1, blocked_event = -1;
    while (finished < grid) {
        while (next_wg < grid && running < resident) {
            M.g[next_wg].started = 1;
            ++next_wg;
            ++running;
        }
        order.clear();
        for (int wg = 0; wg < next_wg; ++wg)
            if (!M.g[wg].ended)
                for (int wv = 0; wv < kWaves; ++wv) order.push_back(wg * kWaves + wv);
        if (seed)
            for (size_t i = order.size(); i > 1; --i) std::swap(order[i - 1], order[next_rand(st) % i]);
        bool progress = false;
        for (int id : order) {
            Group& gr = M.g[id / kWaves];
            const int wv = id % kWaves;
            const int burst = seed ? 1 + (int)(next_rand(st) & 7u) : 1;
            for (int i = 0; i < burst && step(M, gr, wv); ++i) progress = true;
        }
        for (int wg = 0; wg < next_wg; ++wg) {
            Group& gr = M.g[wg];
            if (gr.ended) continue;
            bool all = true;
            for (int wv = 0; wv < kWaves; ++wv) all = all && gr.w[wv].prog[gr.w[wv].pc].ev == kEvEnd;
            if (all) {
                gr.ended = 1;
                --running;
                ++finished;
                progress = true;
            }
        }
        if (!progress) {
            for (int wg = 0; wg < next_wg && blocked_wg < 0; ++wg)
                for (int wv = 0; wv < kWaves; ++wv)
                    if (!M.g[wg].ended && M.g[wg].w[wv].prog[M.g[wg].w[wv].pc].ev != kEvEnd) {
                        blocked_wg = wg;
                        blocked_wave = wv;
                        blocked_event = M.g[wg].w[wv].prog[M.g[wg].w[wv].pc].ev;
                        break;
                    }
            break;
        }
    }
    out->complete = finished == grid ? 1 : 0;
    out->violations = M.violations;
    out->first_violation = M.first_violation;
    out->events = M.events;
    out->blocked_wg = blocked_wg;
    out->blocked_wave = blocked_wave;
    out->blocked_event = blocked_event;
    out->active_experts = M.U;
    out->reserved = 0;
    return MONOMOE_OK;
}
