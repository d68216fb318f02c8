// Host runtime behind include/monomoe.h: plan validation, persistent-grid sizing with an
// occupancy check, workspace ownership and the single-launch forward.
#include "../../include/monomoe.h"
#include "monomoe_internal.h"

#include <hip/hip_ext.h>
#include <cmath>
#include <algorithm>

#include <mutex>
#include <new>
#include <string.h>

using namespace monomoe;

// Kernel choice and LDS layout of a plan.
struct KernelConfig {
    const KernelVariant* var;   // the kernel that runs
    int mt;                     // 1: multi-tile kernel
    int occupancy;
    int lds_dyn;
    int lds_static;
    int naq;
    int nslots;
    int tchunk;                 // single-tile: tokens per pass (T beyond one tile runs in passes)
    int rows, pool, tiles;      // multi-tile: R, quantised-input ring rows, N tiles per slot
};

struct monomoe_plan_s {
    monomoe_shape_t shape;
    int topk;
    int renorm;
    const KernelEntry* kern;
    const KernelVariant* mtv;   // the shape's multi-tile kernel
    const KernelVariant* var;   // the kernel that runs (scheduled ring depth, or multi-tile)
    int device;
    int num_cus;
    int lds_total;              // LDS per workgroup of the device
    int occupancy;
    int grid;
    int lds_dyn;
    int lds_static;
    int naq;
    int nslots;
    int tchunk;   // tokens per pass (T larger than one LDS-resident tile runs in passes)
    int mt;       // multi-tile kernel
    int mt_rows, mt_pool, mt_tiles;
    int general_only;           // schedule: no one-token specialisation
    int up_lb;                  // schedule: gate/up units per deal 2^up_lb (single-tile kernel)
    int down_grid;              // schedule: workgroups with down units (0: the whole grid)
    KernelConfig cfg;           // the configuration above, as chosen for T
    KernelConfig small;         // single-tile configuration for forwards of at most small_T
    int small_T;                //   tokens when cfg is the multi-tile kernel (0: none)
    const float* bias;
    const float* sel_bias;
    int policy;
    float route_scale;
    // workspace (one allocation)
    void* ws;
    size_t ws_bytes;
    uint32_t* ctl;
    uint64_t* logits;
    uint64_t* xq;
    uint64_t* xs;
    uint64_t* act;
    uint64_t* contrib;
};

namespace {

constexpr uint64_t kDefaultSpinTicks = 200000000ull;   // 2 s of the 100 MHz realtime clock

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// The dynamic-LDS limit of a kernel symbol is process-wide state shared by every plan that
// launches it, so it is raised to the most any plan can request (all of the workgroup's LDS
// beyond the kernel's static share) and never lowered: a plan created later with a smaller
// footprint must not invalidate the launches of an earlier, larger one.
hipError_t allow_full_lds(const void* fn, int lds_total, const hipFuncAttributes* attr) {
    return hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize,
                               lds_total - (int)attr->sharedSizeBytes);
}

// Single-tile kernel at ring depth `ring`: the largest token tile (<= kTMax, <= T) whose
// LDS footprint fits, the requantised activation double-buffered when it fits, then as
// many partial-sum slots as the rest of the LDS holds (more slots let the compute
// wavefronts run further ahead of the helper's epilogues).  Every ring depth must fit, so
// schedules can switch.
// Host arithmetic of the layouts and of residency (no device call), shared by plan
// creation and monomoe_layout.
//
// Single-tile kernel, T tokens, lds_cap bytes of dynamic LDS: the largest token tile (a
// pass) that fits with one act buffer and the minimum of hand-off slots, the act double
// buffered when that fits too, then as many slots (a power of two) as fit.
int single_layout(int H, int I, int T, int lds_cap, KernelConfig* k) {
    int Tl = std::min(std::max(T, 1), kTMax);
    while (Tl > 1 && lds_dynamic_bytes(H, I, Tl, 1, kSlotsMin) > lds_cap) --Tl;
    k->tchunk = Tl;
    k->naq = lds_dynamic_bytes(H, I, Tl, 2, kSlotsMin) <= lds_cap ? 2 : 1;
    k->nslots = kSlotsMin;
    while (k->nslots < kSlotsMax && lds_dynamic_bytes(H, I, Tl, k->naq, k->nslots * 2) <= lds_cap) k->nslots *= 2;
    k->lds_dyn = lds_dynamic_bytes(H, I, Tl, k->naq, k->nslots);
    return k->lds_dyn > lds_cap ? MONOMOE_ERR_UNSUPPORTED : MONOMOE_OK;
}

// Multi-tile kernel: the largest segment size R (<= T, <= group_cap when nonzero) whose
// LDS layout fits, then as many quantised-input ring rows as the rest holds.  Segments
// per forward are bounded by min(E, T*k) + ceil(T*k / R), which must fit the kernel's
// segment queue.
int multi_layout(int H, int I, int T, int E, int topk, int group_cap, int lds_cap, KernelConfig* k) {
    T = std::max(T, 1);
    int R = std::min(T, kTLimit);
    if (group_cap > 0) R = std::min(R, group_cap);
    for (; R >= 1; --R) {
        k->tiles = (R + 15) / 16;
        if (mt_region_bytes(H, I, R, R) + mt_partials_bytes(kSlotsMin, k->tiles) <= lds_cap) break;
    }
    if (R < 1) return MONOMOE_ERR_UNSUPPORTED;
    k->rows = R;
    k->pool = R;
    while (k->pool < 1024 && mt_region_bytes(H, I, k->pool + 1, R) + mt_partials_bytes(kSlotsMin, k->tiles) <= lds_cap)
        ++k->pool;
    const int pairs = T * topk;
    if (std::min(E, pairs) + (pairs + R - 1) / R > kQMax) return MONOMOE_ERR_UNSUPPORTED;
    k->naq = 2;
    k->nslots = kSlotsMin;
    k->tchunk = T;
    k->lds_dyn = mt_region_bytes(H, I, k->pool, R) + mt_partials_bytes(k->nslots, k->tiles);
    return MONOMOE_OK;
}

// A persistent grid waits across workgroups, so all of its workgroups must be resident at
// once: grid <= num_cus * occupancy (workgroups per CU the layout allows).
int residency(int occupancy, int grid, int num_cus) {
    return (occupancy < 1 || (int64_t)grid > (int64_t)num_cus * occupancy) ? MONOMOE_ERR_OCCUPANCY : MONOMOE_OK;
}

int config_single(const monomoe_plan_s* pl, int ring, KernelConfig* c) {
    const monomoe_shape_t& s = pl->shape;
    const KernelVariant* var = nullptr;
    for (const KernelVariant& v : pl->kern->v)
        if (v.ring == ring) var = &v;
    if (!var) return MONOMOE_ERR_INVALID;
    hipFuncAttributes attr;
    if (hipFuncGetAttributes(&attr, var->fn) != hipSuccess) return MONOMOE_ERR_HIP;
    KernelConfig k{};
    k.var = var;
    k.lds_static = (int)attr.sharedSizeBytes;
    const int lr = single_layout(s.H, s.I, s.T, pl->lds_total - k.lds_static, &k);
    if (lr != MONOMOE_OK) return lr;
    k.occupancy = 0;
    for (const KernelVariant& v : pl->kern->v) {
        for (const void* fn : {v.fn, v.fn1}) {   // the kernel and its one-token specialisation
            if (!fn) continue;
            hipFuncAttributes va;
            int o = 0;
            if (hipFuncGetAttributes(&va, fn) != hipSuccess || allow_full_lds(fn, pl->lds_total, &va) != hipSuccess ||
                hipOccupancyMaxActiveBlocksPerMultiprocessor(&o, fn, kThreads, (size_t)k.lds_dyn) != hipSuccess)
                return MONOMOE_ERR_HIP;
            if ((int)va.sharedSizeBytes + k.lds_dyn > pl->lds_total) return MONOMOE_ERR_UNSUPPORTED;
            if (residency(o, pl->num_cus, pl->num_cus) != MONOMOE_OK) return MONOMOE_ERR_OCCUPANCY;
            if (&v == var) k.occupancy = k.occupancy ? std::min(k.occupancy, o) : o;
        }
    }
    *c = k;
    return MONOMOE_OK;
}

// Multi-tile kernel configuration of a plan (layout: multi_layout).
int config_multi(const monomoe_plan_s* pl, int group_cap, KernelConfig* c) {
    const monomoe_shape_t& s = pl->shape;
    if (!pl->mtv) return MONOMOE_ERR_UNSUPPORTED;
    hipFuncAttributes attr;
    if (hipFuncGetAttributes(&attr, pl->mtv->fn) != hipSuccess) return MONOMOE_ERR_HIP;
    KernelConfig k{};
    k.var = pl->mtv;
    k.mt = 1;
    k.lds_static = (int)attr.sharedSizeBytes;
    const int lr = multi_layout(s.H, s.I, s.T, s.E, pl->topk, group_cap, pl->lds_total - k.lds_static, &k);
    if (lr != MONOMOE_OK) return lr;
    int o = 0;
    if (allow_full_lds(k.var->fn, pl->lds_total, &attr) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&o, k.var->fn, kThreads, (size_t)k.lds_dyn) != hipSuccess)
        return MONOMOE_ERR_HIP;
    if (residency(o, pl->num_cus, pl->num_cus) != MONOMOE_OK) return MONOMOE_ERR_OCCUPANCY;
    k.occupancy = o;
    *c = k;
    return MONOMOE_OK;
}

// Kernel for a request: MONOMOE_KERNEL_AUTO takes the single-tile kernel while T fits
// its tile and the multi-tile kernel beyond (token passes if that cannot be configured).
// Where the down projection is sliced (I > 2048) the multi-tile kernel runs at every T:
// the single-tile kernel requantises each expert's whole activation row (I = 14336) into
// LDS before its first down task, which the sliced kernel splits over the slices
// (measured on the 4096x14336 layer: 272 vs 313 us at T = 8, 321 vs 646 us at T = 16; at
// T = 1 the two kernels are within 2% of each other).
// When the automatic choice is the multi-tile kernel for the plan's T, *small receives the
// single-tile configuration and *small_T the token counts up to which a forward with fewer
// tokens (monomoe_forward_tokens) takes it instead (0: every T takes *c).
int configure(const monomoe_plan_s* pl, int kernel, int ring, int group_cap, KernelConfig* c,
              KernelConfig* small, int* small_T) {
    *small_T = 0;
    if (kernel == MONOMOE_KERNEL_MULTI) {
        if (ring != 0 && ring != pl->mtv->ring) return MONOMOE_ERR_INVALID;
        return config_multi(pl, group_cap, c);
    }
    const int r = ring == 0 ? pl->kern->ring_default : ring;
    const int rc = config_single(pl, r, c);
    const int ib = pl->shape.I / 128;
    const bool sliced = mt_slice_blocks(ib) != ib;
    if (rc != MONOMOE_OK || kernel == MONOMOE_KERNEL_SINGLE || (pl->shape.T <= c->tchunk && !sliced)) return rc;
    if (ring != 0 && ring != pl->mtv->ring) return MONOMOE_OK;   // that depth exists in the single-tile kernel only
    KernelConfig m;
    if (config_multi(pl, group_cap, &m) == MONOMOE_OK) {
        // forwards that fit the single-tile kernel's tile stay on it; with a sliced down
        // projection only forwards of one token do (its one-token specialisation is faster
        // there, the multi-tile kernel from two tokens on)
        *small = *c;
        *small_T = sliced ? 1 : c->tchunk;
        *c = m;
    }
    return MONOMOE_OK;
}

void apply_config(monomoe_plan_s* pl, const KernelConfig& c, const KernelConfig& small, int small_T) {
    pl->cfg = c;
    pl->small = small;
    pl->small_T = small_T;
    pl->var = c.var;
    pl->mt = c.mt;
    pl->occupancy = c.occupancy;
    pl->lds_dyn = c.lds_dyn;
    pl->lds_static = c.lds_static;
    pl->naq = c.naq;
    pl->nslots = c.nslots;
    pl->tchunk = c.tchunk;
    pl->mt_rows = c.rows;
    pl->mt_pool = c.pool;
    pl->mt_tiles = c.tiles;
}

int zero_workspace(monomoe_plan_s* pl) {
    if (hipMemset(pl->ws, 0, pl->ws_bytes) != hipSuccess) return MONOMOE_ERR_HIP;
    if (hipDeviceSynchronize() != hipSuccess) return MONOMOE_ERR_HIP;
    return MONOMOE_OK;
}

// Kernel configuration and persistent grid of a new plan (shape, topk, renorm set) on
// device dev: one workgroup per compute unit, the automatic kernel choice.
int configure_plan(monomoe_plan_s* pl, int dev, int num_cus, int lds_total) {
    pl->device = dev;
    pl->num_cus = num_cus;
    pl->lds_total = lds_total;
    KernelConfig cfg{}, small{};
    int small_T = 0;
    const int cr = configure(pl, MONOMOE_KERNEL_AUTO, 0, 0, &cfg, &small, &small_T);
    if (cr != MONOMOE_OK) return cr;
    apply_config(pl, cfg, small, small_T);
    pl->grid = pl->num_cus;   // one resident workgroup per CU
    if (pl->grid > kGridMax) return MONOMOE_ERR_UNSUPPORTED;
    return MONOMOE_OK;
}

// Workspace layout: control words | logits | quantised input (codes, scales) | act |
// contrib, sized for one launch over every token of the plan and for the multi-tile
// kernel's down slices.  Returns the total size; with a base address it also sets the
// plan's workspace pointers.
size_t layout_workspace(monomoe_plan_s* pl, uint8_t* base) {
    const monomoe_shape_t& s = pl->shape;
    const int T = std::max(s.T, 1), topk = pl->topk;
    const int nsl = (s.I / 128) / mt_slice_blocks(s.I / 128);
    size_t off = 0;
    const size_t o_ctl = off;    off = align_up(off + sizeof(uint32_t) * ctl_words(), 256);
    const size_t o_log = off;    off = align_up(off + sizeof(uint64_t) * (size_t)T * s.E, 256);
    const size_t o_xq = off;     off = align_up(off + sizeof(uint64_t) * (size_t)T * s.H / 4, 256);
    const size_t o_xs = off;     off = align_up(off + sizeof(uint64_t) * (size_t)T * s.H / 128, 256);
    const size_t o_act = off;    off = align_up(off + sizeof(uint64_t) * (size_t)T * topk * s.I, 256);
    const size_t o_out = off;    off = align_up(off + sizeof(uint64_t) * (size_t)T * topk * nsl * s.H, 256);
    if (base) {
        pl->ctl = reinterpret_cast<uint32_t*>(base + o_ctl);
        pl->logits = reinterpret_cast<uint64_t*>(base + o_log);
        pl->xq = reinterpret_cast<uint64_t*>(base + o_xq);
        pl->xs = reinterpret_cast<uint64_t*>(base + o_xs);
        pl->act = reinterpret_cast<uint64_t*>(base + o_act);
        pl->contrib = reinterpret_cast<uint64_t*>(base + o_out);
    }
    return off;
}

// Shape and routing checks shared by monomoe_plan and the allocation-free forward.
int check_shape(const monomoe_shape_t& s, int topk) {
    if (s.T < 0 || s.H <= 0 || s.I <= 0 || s.E <= 0) return MONOMOE_ERR_INVALID;
    if (s.H % 128 || s.I % 128) return MONOMOE_ERR_INVALID;
    if (topk < 1 || topk > s.E) return MONOMOE_ERR_INVALID;
    if (s.T > kTLimit || s.E > kEMax || topk > kKMax) return MONOMOE_ERR_UNSUPPORTED;
    if (!find_kernel(s.H, s.I)) return MONOMOE_ERR_UNSUPPORTED;
    return MONOMOE_OK;
}

// One forward of T tokens (0 <= T <= the plan's T) with the plan's configuration for T.
int launch(monomoe_plan_t plan, int T, const void* x, const void* router_w, const void* w13, const float* w13_scale,
           const void* w2, const float* w2_scale, void* out, const monomoe_debug_t* dbg, hipStream_t stream,
           hipEvent_t ev_start = nullptr, hipEvent_t ev_stop = nullptr) {
    if (!plan) return MONOMOE_ERR_INVALID;
    const monomoe_shape_t& s = plan->shape;
    if (T < 0 || T > s.T) return MONOMOE_ERR_INVALID;
    if (T == 0) return MONOMOE_OK;
    const KernelConfig& cf = (T <= plan->small_T) ? plan->small : plan->cfg;
    if (!x || !router_w || !w13 || !w13_scale || !w2 || !w2_scale || !out) return MONOMOE_ERR_INVALID;
    if (!aligned16(x) || !aligned16(router_w) || !aligned16(w13) || !aligned16(w2) || !aligned16(out) ||
        !aligned16(w13_scale) || !aligned16(w2_scale))
        return MONOMOE_ERR_INVALID;

    KParams p;
    memset(&p, 0, sizeof p);
    p.x = static_cast<const uint16_t*>(x);
    p.rw = static_cast<const uint16_t*>(router_w);
    p.bias = plan->bias;
    p.sel_bias = plan->sel_bias;
    p.policy = plan->policy;
    p.route_scale = plan->route_scale;
    p.w13 = static_cast<const uint8_t*>(w13);
    p.w13s = w13_scale;
    p.w2 = static_cast<const uint8_t*>(w2);
    p.w2s = w2_scale;
    p.out = static_cast<uint16_t*>(out);
    p.ctl = plan->ctl;
    p.logits = plan->logits;
    p.xqw = plan->xq;
    p.xsw = plan->xs;
    p.act = plan->act;
    p.contrib = plan->contrib;
    p.spin_limit = kDefaultSpinTicks;
    if (dbg) {
        if ((dbg->topk_ids == nullptr) != (dbg->topk_w == nullptr)) return MONOMOE_ERR_INVALID;
        if ((dbg->xq == nullptr) != (dbg->xs == nullptr)) return MONOMOE_ERR_INVALID;
        if ((dbg->aq == nullptr) != (dbg->as == nullptr)) return MONOMOE_ERR_INVALID;
        if ((dbg->topk_ids_in == nullptr) != (dbg->topk_w_in == nullptr)) return MONOMOE_ERR_INVALID;
        if (dbg->jitter_seed > 0xFFFFu) return MONOMOE_ERR_INVALID;
#ifndef MONOMOE_RACE_PERTURB
        if (dbg->jitter_seed != 0) return MONOMOE_ERR_UNSUPPORTED;   // the perturbation build's hook
#endif
        p.d_ids = dbg->topk_ids;
        p.d_w = dbg->topk_w;
        p.d_xq = dbg->xq;
        p.d_xs = dbg->xs;
        p.d_act = dbg->act;
        p.d_aq = dbg->aq;
        p.d_as = dbg->as;
        p.d_out = dbg->out_f32;
        p.inj_ids = dbg->topk_ids_in;
        p.inj_w = dbg->topk_w_in;
        p.stamps = dbg->stamps;
        if (dbg->spin_limit_ticks) p.spin_limit = dbg->spin_limit_ticks;
        p.fail_flag = dbg->fail_flag != 0;
        p.jitter = (uint16_t)dbg->jitter_seed;
    }
    p.E = s.E;
    p.k = plan->topk;
    p.renorm = plan->renorm;
    p.naq = (int16_t)cf.naq;
    p.nslots = (int16_t)cf.nslots;
    p.up_lb = (uint8_t)plan->up_lb;
    p.dn_grid = (uint16_t)(plan->down_grid ? plan->down_grid : plan->grid);
    p.mt_rows = (uint8_t)cf.rows;
    p.mt_tiles = (uint8_t)cf.tiles;
    p.mt_pool = (uint16_t)cf.pool;

    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess || cur != plan->device) return MONOMOE_ERR_INVALID;
    // one launch per pass of at most tchunk tokens (one pass when T fits one tile); each
    // pass sees its rows of every token-indexed buffer
    const int K = plan->topk, H = s.H, I = s.I, tc = cf.mt ? T : cf.tchunk;
    for (int t0 = 0; t0 < T; t0 += tc) {
        KParams q = p;
        q.T = std::min(tc, T - t0);
        q.x = p.x + (size_t)t0 * H;
        q.out = p.out + (size_t)t0 * H;
        if (p.d_ids) q.d_ids = p.d_ids + (size_t)t0 * K;
        if (p.d_w) q.d_w = p.d_w + (size_t)t0 * K;
        if (p.d_xq) q.d_xq = p.d_xq + (size_t)t0 * H;
        if (p.d_xs) q.d_xs = p.d_xs + (size_t)t0 * (H / 128);
        if (p.d_act) q.d_act = p.d_act + (size_t)t0 * K * I;
        if (p.d_aq) q.d_aq = p.d_aq + (size_t)t0 * K * I;
        if (p.d_as) q.d_as = p.d_as + (size_t)t0 * K * (I / 128);
        if (p.d_out) q.d_out = p.d_out + (size_t)t0 * H;
        if (p.inj_ids) q.inj_ids = p.inj_ids + (size_t)t0 * K;
        if (p.inj_w) q.inj_w = p.inj_w + (size_t)t0 * K;
        const bool first = t0 == 0, last = t0 + tc >= T;
        // a pass of one token runs the one-token specialisation (not under the timeout test hook)
        const bool one = q.T == 1 && !q.fail_flag && cf.var->fn1 != nullptr && !plan->general_only;
        if (ev_start || ev_stop) {
            // the dispatch itself records the events (the first pass's begin, the last
            // pass's end), not the stream
            void* args[] = {&q};
            if (hipExtLaunchKernel(one ? cf.var->fn1 : cf.var->fn, dim3(plan->grid), dim3(kThreads), args,
                                   (size_t)cf.lds_dyn, stream, first ? ev_start : nullptr, last ? ev_stop : nullptr,
                                   0) != hipSuccess)
                return MONOMOE_ERR_HIP;
        } else {
            (one ? cf.var->launch1 : cf.var->launch)(q, plan->grid, (size_t)cf.lds_dyn, stream);
        }
        if (hipGetLastError() != hipSuccess) return MONOMOE_ERR_HIP;
    }
    return MONOMOE_OK;
}

}  // namespace

// ------------------------------------------------------------------------------------
// Allocation-free forward (monomoe_forward_noalloc): the workspace lives in one file-scope
// device array instead of a plan's hipMalloc'd buffer.
// ------------------------------------------------------------------------------------
constexpr size_t kNoAllocScratchBytes = size_t(32) << 20;   // the largest workspace it serves

// One copy per GPU the library runs on, held until the process ends.  Static storage, so it
// is zero when the code object is loaded: every launch epoch 0 and the status word clear,
// the state the tagged-exchange protocol starts from.  Host code must never pass this name
// to a kernel (on the host it is a stand-in, not a device address): the device address is
// taken once per device with hipGetSymbolAddress and kept in g_scratch_dev.
static __device__ __align__(256) uint8_t scratch[kNoAllocScratchBytes];

namespace {

constexpr int kNoAllocDevices = 64;
constexpr int kNoAllocCache = 8;

struct NoAllocEntry {
    int valid, dev, topk, renorm;
    monomoe_shape_t shape;
    monomoe_plan_s plan;   // configuration and workspace pointers into the device's scratch
};

std::mutex g_noalloc_mu;
uint8_t* g_scratch_dev[kNoAllocDevices];   // device address of `scratch`, per device
NoAllocEntry g_noalloc_cache[kNoAllocCache];
int g_noalloc_next = 0;

// Reports the device status of the launch before it (MONOMOE_OK, MONOMOE_ERR_TIMEOUT or
// MONOMOE_ERR_INVALID for a rejected expert id) into *out when out is not null, and clears
// the status word, so one failed call does not fail every later one.
__global__ void noalloc_status(uint32_t* word, int32_t* out) {
    if (threadIdx.x != 0) return;
    const uint32_t st = __hip_atomic_load(word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (out) *out = st == kDevOk ? MONOMOE_OK : (st == kDevTimeout ? MONOMOE_ERR_TIMEOUT : MONOMOE_ERR_INVALID);
    if (st != kDevOk) __hip_atomic_store(word, (uint32_t)kDevOk, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The configuration of (device, shape, topk, renorm) with its workspace laid out in the
// device's scratch; computed on first use (set-up of the device included) and cached.
int noalloc_plan(int dev, const monomoe_shape_t& s, int topk, int renorm, monomoe_plan_s* out) {
    std::lock_guard<std::mutex> lock(g_noalloc_mu);
    if (!g_scratch_dev[dev]) {
        void* ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return MONOMOE_ERR_HIP;
        g_scratch_dev[dev] = static_cast<uint8_t*>(ptr);
    }
    for (const NoAllocEntry& c : g_noalloc_cache) {
        if (c.valid && c.dev == dev && c.topk == topk && c.renorm == renorm && c.shape.T == s.T && c.shape.H == s.H &&
            c.shape.E == s.E && c.shape.I == s.I) {
            *out = c.plan;
            return MONOMOE_OK;
        }
    }
    monomoe_plan_s pl{};
    pl.shape = s;
    pl.topk = topk;
    pl.renorm = renorm ? 1 : 0;
    pl.kern = find_kernel(s.H, s.I);
    pl.mtv = find_mt_kernel(s.H, s.I);
    pl.policy = MONOMOE_ROUTING_SOFTMAX;
    pl.route_scale = 1.0f;
    int cus = 0, lds = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipDeviceGetAttribute(&lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess)
        return MONOMOE_ERR_HIP;
    const int cr = configure_plan(&pl, dev, cus, lds);
    if (cr != MONOMOE_OK) return cr;
    const size_t need = layout_workspace(&pl, nullptr);
    if (need > kNoAllocScratchBytes) return MONOMOE_ERR_UNSUPPORTED;
    pl.ws = g_scratch_dev[dev];
    pl.ws_bytes = need;
    layout_workspace(&pl, g_scratch_dev[dev]);
    NoAllocEntry& slot = g_noalloc_cache[g_noalloc_next];
    g_noalloc_next = (g_noalloc_next + 1) % kNoAllocCache;
    slot.valid = 1;
    slot.dev = dev;
    slot.topk = topk;
    slot.renorm = renorm ? 1 : 0;
    slot.shape = s;
    slot.plan = pl;
    *out = pl;
    return MONOMOE_OK;
}

}  // namespace

extern "C" {

int monomoe_forward_noalloc(const monomoe_shape_t* shape, int topk, int renorm, const float* bias, const void* x,
                            const void* router_w, const void* w13, const float* w13_scale, const void* w2,
                            const float* w2_scale, void* out, int32_t* status, hipStream_t stream) {
    if (!shape) return MONOMOE_ERR_INVALID;
    const int sc = check_shape(*shape, topk);
    if (sc != MONOMOE_OK) return sc;
    if ((bias && !aligned16(bias)) || (reinterpret_cast<uintptr_t>(status) & 3u)) return MONOMOE_ERR_INVALID;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return MONOMOE_ERR_HIP;
    if (dev < 0 || dev >= kNoAllocDevices) return MONOMOE_ERR_UNSUPPORTED;
    monomoe_plan_s pl;
    const int pr = noalloc_plan(dev, *shape, topk, renorm, &pl);
    if (pr != MONOMOE_OK) return pr;
    pl.bias = bias;
    const int rc = launch(&pl, shape->T, x, router_w, w13, w13_scale, w2, w2_scale, out, nullptr, stream);
    if (rc != MONOMOE_OK || shape->T == 0) return rc;
    hipLaunchKernelGGL(noalloc_status, dim3(1), dim3(64), 0, stream, pl.ctl + kCtlStatus, status);
    if (hipGetLastError() != hipSuccess) return MONOMOE_ERR_HIP;
    return MONOMOE_OK;
}

int monomoe_supported_shape(int32_t H, int32_t I) { return find_kernel(H, I) ? 1 : 0; }

const char* monomoe_status_string(int status) {
    switch (status) {
        case MONOMOE_OK: return "ok";
        case MONOMOE_ERR_INVALID: return "invalid argument";
        case MONOMOE_ERR_UNSUPPORTED: return "unsupported shape";
        case MONOMOE_ERR_OCCUPANCY: return "persistent grid cannot be resident";
        case MONOMOE_ERR_HIP: return "HIP runtime error";
        case MONOMOE_ERR_TIMEOUT: return "device readiness wait timed out";
        default: return "unknown status";
    }
}

int monomoe_plan(const monomoe_shape_t* shape, int topk, int renorm, monomoe_plan_t* plan_out) {
    if (!shape || !plan_out) return MONOMOE_ERR_INVALID;
    const monomoe_shape_t s = *shape;
    const int sc = check_shape(s, topk);
    if (sc != MONOMOE_OK) return sc;
    const KernelEntry* kern = find_kernel(s.H, s.I);

    monomoe_plan_s* pl = new (std::nothrow) monomoe_plan_s();
    if (!pl) return MONOMOE_ERR_HIP;
    pl->shape = s;
    pl->topk = topk;
    pl->renorm = renorm ? 1 : 0;
    pl->kern = kern;
    pl->mtv = find_mt_kernel(s.H, s.I);
    pl->bias = nullptr;
    pl->sel_bias = nullptr;
    pl->policy = MONOMOE_ROUTING_SOFTMAX;
    pl->route_scale = 1.0f;

    int dev = 0;
    hipDeviceProp_t prop;
    if (hipGetDevice(&dev) != hipSuccess || hipGetDeviceProperties(&prop, dev) != hipSuccess) {
        delete pl;
        return MONOMOE_ERR_HIP;
    }
    const int cr = configure_plan(pl, dev, prop.multiProcessorCount, (int)prop.sharedMemPerBlock);
    if (cr != MONOMOE_OK) {
        delete pl;
        return cr;
    }
    pl->ws_bytes = layout_workspace(pl, nullptr);
    if (hipMalloc(&pl->ws, pl->ws_bytes) != hipSuccess) {
        delete pl;
        return MONOMOE_ERR_HIP;
    }
    layout_workspace(pl, static_cast<uint8_t*>(pl->ws));
    const int zr = zero_workspace(pl);
    if (zr != MONOMOE_OK) {
        (void)hipFree(pl->ws);
        delete pl;
        return zr;
    }
    *plan_out = pl;
    return MONOMOE_OK;
}

void monomoe_plan_destroy(monomoe_plan_t plan) {
    if (!plan) return;
    if (plan->ws) (void)hipFree(plan->ws);
    delete plan;
}

int monomoe_plan_set_router_bias(monomoe_plan_t plan, const float* bias) {
    if (!plan) return MONOMOE_ERR_INVALID;
    if (bias && !aligned16(bias)) return MONOMOE_ERR_INVALID;
    plan->bias = bias;
    return MONOMOE_OK;
}

static_assert(MONOMOE_ROUTING_SOFTMAX == kRouteSoftmax && MONOMOE_ROUTING_SIGMOID_BIAS == kRouteSigmoidBias,
              "routing policy values");
int monomoe_plan_set_routing(monomoe_plan_t plan, int policy, const float* sel_bias, float scale) {
    if (!plan) return MONOMOE_ERR_INVALID;
    if (policy == MONOMOE_ROUTING_SOFTMAX) {
        if (sel_bias || scale != 1.0f) return MONOMOE_ERR_INVALID;
    } else if (policy == MONOMOE_ROUTING_SIGMOID_BIAS) {
        if (!(scale > 0.0f) || !(scale < INFINITY)) return MONOMOE_ERR_INVALID;
        if (sel_bias && !aligned16(sel_bias)) return MONOMOE_ERR_INVALID;
    } else {
        return MONOMOE_ERR_INVALID;
    }
    plan->policy = policy;
    plan->sel_bias = sel_bias;
    plan->route_scale = scale;
    return MONOMOE_OK;
}

int monomoe_plan_set_schedule(monomoe_plan_t plan, const monomoe_schedule_t* sched) {
    if (!plan || !sched) return MONOMOE_ERR_INVALID;
    if (sched->kernel < MONOMOE_KERNEL_AUTO || sched->kernel > MONOMOE_KERNEL_MULTI) return MONOMOE_ERR_INVALID;
    if (sched->group_tokens < 0 || sched->group_tokens > kTLimit) return MONOMOE_ERR_INVALID;
    if (sched->ring != 0 && sched->ring != kRings[0] && sched->ring != kRings[1]) return MONOMOE_ERR_INVALID;
    if (sched->general_only != 0 && sched->general_only != 1) return MONOMOE_ERR_INVALID;
    int up_lb = 0;
    while (up_lb < kUpBlockLogMax && (1 << up_lb) < sched->up_block) ++up_lb;
    if (sched->up_block < 0 || (sched->up_block > 0 && (1 << up_lb) != sched->up_block)) return MONOMOE_ERR_INVALID;
    if (sched->down_grid < 0) return MONOMOE_ERR_INVALID;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev != plan->device) return MONOMOE_ERR_INVALID;
    KernelConfig cfg{}, small{};
    int small_T = 0;
    const int cr = configure(plan, sched->kernel, sched->ring, sched->group_tokens, &cfg, &small, &small_T);
    if (cr != MONOMOE_OK) return cr;
    const int grid = sched->grid == 0 ? plan->num_cus : sched->grid;
    if (grid < 1 || grid > plan->num_cus * cfg.occupancy || grid > kGridMax) return MONOMOE_ERR_INVALID;
    if (sched->down_grid > grid) return MONOMOE_ERR_INVALID;
    if (small_T > 0 && grid > plan->num_cus * small.occupancy) small_T = 0;
    // the launch epochs are per workgroup: a new grid starts from a clean workspace
    if (grid != plan->grid) {
        if (hipDeviceSynchronize() != hipSuccess) return MONOMOE_ERR_HIP;
        const int zr = zero_workspace(plan);
        if (zr != MONOMOE_OK) return zr;
    }
    plan->grid = grid;
    plan->general_only = sched->general_only;
    plan->up_lb = up_lb;
    plan->down_grid = sched->down_grid == grid ? 0 : sched->down_grid;
    apply_config(plan, cfg, small, small_T);
    return MONOMOE_OK;
}

int monomoe_forward(monomoe_plan_t plan, const void* x, const void* router_w, const void* w13,
                    const float* w13_scale, const void* w2, const float* w2_scale, void* out, hipStream_t stream) {
    if (!plan) return MONOMOE_ERR_INVALID;
    return launch(plan, plan->shape.T, x, router_w, w13, w13_scale, w2, w2_scale, out, nullptr, stream);
}

int monomoe_forward_tokens(monomoe_plan_t plan, int32_t T, const void* x, const void* router_w, const void* w13,
                           const float* w13_scale, const void* w2, const float* w2_scale, void* out,
                           hipStream_t stream) {
    return launch(plan, T, x, router_w, w13, w13_scale, w2, w2_scale, out, nullptr, stream);
}

int monomoe_forward_timed(monomoe_plan_t plan, const void* x, const void* router_w, const void* w13,
                          const float* w13_scale, const void* w2, const float* w2_scale, void* out,
                          hipEvent_t start, hipEvent_t stop, hipStream_t stream) {
    if (!plan || !start || !stop) return MONOMOE_ERR_INVALID;
    return launch(plan, plan->shape.T, x, router_w, w13, w13_scale, w2, w2_scale, out, nullptr, stream, start, stop);
}

int monomoe_forward_debug(monomoe_plan_t plan, const void* x, const void* router_w, const void* w13,
                          const float* w13_scale, const void* w2, const float* w2_scale, void* out,
                          const monomoe_debug_t* dbg, hipStream_t stream) {
    if (!plan) return MONOMOE_ERR_INVALID;
    return launch(plan, plan->shape.T, x, router_w, w13, w13_scale, w2, w2_scale, out, dbg, stream);
}

int monomoe_plan_status(monomoe_plan_t plan) {
    if (!plan) return MONOMOE_ERR_INVALID;
    if (hipDeviceSynchronize() != hipSuccess) return MONOMOE_ERR_HIP;
    uint32_t st = 0;
    if (hipMemcpy(&st, plan->ctl + kCtlStatus, sizeof st, hipMemcpyDeviceToHost) != hipSuccess) return MONOMOE_ERR_HIP;
    if (st == kDevOk) return MONOMOE_OK;
    if (st == kDevTimeout) return MONOMOE_ERR_TIMEOUT;
    return MONOMOE_ERR_INVALID;
}

int monomoe_plan_reset(monomoe_plan_t plan) {
    if (!plan) return MONOMOE_ERR_INVALID;
    if (hipDeviceSynchronize() != hipSuccess) return MONOMOE_ERR_HIP;
    return zero_workspace(plan);
}

int monomoe_layout(const monomoe_shape_t* shape, int topk, int kernel, int lds_total, int lds_static,
                   int occupancy, int grid, int num_cus, monomoe_layout_t* out) {
    if (!shape || !out) return MONOMOE_ERR_INVALID;
    const monomoe_shape_t s = *shape;
    const int sc = check_shape(s, topk);
    if (sc != MONOMOE_OK) return sc;
    if (kernel != MONOMOE_KERNEL_SINGLE && kernel != MONOMOE_KERNEL_MULTI) return MONOMOE_ERR_INVALID;
    if (lds_static < 0 || lds_total <= lds_static || occupancy < 0 || grid < 0 || num_cus < 1) return MONOMOE_ERR_INVALID;
    KernelConfig k{};
    const int lr = kernel == MONOMOE_KERNEL_SINGLE ? single_layout(s.H, s.I, s.T, lds_total - lds_static, &k)
                                                   : multi_layout(s.H, s.I, s.T, s.E, topk, 0, lds_total - lds_static, &k);
    if (lr != MONOMOE_OK) return lr;
    out->tokens_per_pass = k.tchunk;
    out->group_tokens = kernel == MONOMOE_KERNEL_MULTI ? k.rows : 0;
    out->act_buffers = k.naq;
    out->handoff_slots = k.nslots;
    out->lds_bytes = k.lds_dyn;
    return residency(occupancy, grid == 0 ? num_cus : grid, num_cus);
}

int monomoe_plan_info(monomoe_plan_t plan, monomoe_plan_info_t* info) {
    if (!plan || !info) return MONOMOE_ERR_INVALID;
    // the configuration a forward of the plan's T runs (the single-tile one when the
    // multi-tile plan hands forwards of up to small_T tokens to it)
    const KernelConfig& c = plan->shape.T <= plan->small_T ? plan->small : plan->cfg;
    info->grid = plan->grid;
    info->block = kThreads;
    info->lds_bytes = c.lds_dyn + c.lds_static;
    info->occupancy = c.occupancy;
    info->num_cus = plan->num_cus;
    info->workspace_bytes = (int64_t)plan->ws_bytes;
    // scratch of every kernel the plan may launch (and the one-token specialisations)
    info->scratch_bytes = 0;
    const KernelVariant* vars[2] = {plan->cfg.var, plan->small_T > 0 ? plan->small.var : nullptr};
    for (const KernelVariant* v : vars) {
        if (!v) continue;
        for (const void* fn : {v->fn, v->fn1}) {
            hipFuncAttributes attr;
            if (!fn || info->scratch_bytes < 0) continue;
            info->scratch_bytes = hipFuncGetAttributes(&attr, fn) == hipSuccess
                                      ? std::max(info->scratch_bytes, (int32_t)attr.localSizeBytes) : -1;
        }
    }
    info->ring = c.var->ring;
    info->tokens_per_pass = c.tchunk;
    info->multi_tile = c.mt;
    info->group_tokens = c.mt ? c.rows : 0;
    info->down_slices = c.mt ? (plan->shape.I / 128) / mt_slice_blocks(plan->shape.I / 128) : 1;
    info->up_block = 1 << plan->up_lb;
    info->down_grid = plan->down_grid ? plan->down_grid : plan->grid;
    return MONOMOE_OK;
}

}  // extern "C"
