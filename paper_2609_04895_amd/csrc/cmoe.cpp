// cmoe.cpp - host side of the C ABI declared in include/cmoe.h: validation,
// buffer carving, the per-token launch sequence on the main and side streams,
// counters, inspection and kernel timing.
//
// Launch sequence of one token (layers in causal order; "refining modes" are
// the full and Spatio-only modes, which have a Spatio Router):
//   [refining mode, t >= 1, R > 0] main: cache step refining layer 0 from the
//       previous token's last-layer Spatio prediction; side: fill (proactive)
//   for each layer l:
//     main: router GEMV(l)
//     main: [wait for the proactive fill of l] cache step(l): access, retention,
//           counters, buckets; in a refining mode also refinement of layer l + 1
//     main: fill(l, demand)  -- gates the FFN of this layer
//     side: [refining mode] fill(l + 1, proactive), overlapping the FFN of l
//     main: expert gate/up(l), expert down(l), combine(l)
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/cmoe.h"
#include "cmoe_internal.h"

using cmoe::FillArgs;
using cmoe::Layout;
using cmoe::StepArgs;

// Per-step scratch of cmoe_step_noalloc, for callers that cannot allocate a
// workspace: one array per GPU, loaded with the library and held until the
// process ends.  In host code `scratch` names a host-side stand-in, never the
// device memory: the device address comes from hipGetSymbolAddress, taken once
// per device at cmoe_init with that device current.
constexpr size_t kScratchBytes = size_t(64) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

thread_local std::string g_err;

std::mutex g_scratch_mu;
std::vector<void*> g_scratch_ptr;  // device address of `scratch` on each device, once resolved

// The device address of the scratch array on the current device `dev`.
hipError_t scratch_on_device(int dev, void** out) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (dev >= (int)g_scratch_ptr.size()) g_scratch_ptr.resize(dev + 1, nullptr);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}

cmoe_status fail(cmoe_status st, const std::string& msg) {
    g_err = msg;
    return st;
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

enum KernelId { KID_ROUTER = 0, KID_CACHE = 1, KID_FILL = 2, KID_UP = 3, KID_DOWN = 4, KID_COMBINE = 5 };

struct Derived {
    int NW, n_r, n_slots, nsplit, rdk, zstride;
    int rounds;        // FFN rounds per layer step: more than one only for an arena smaller than the union
    int iT, iS;        // router slots of the Temporal / Spatio Router, -1 if not used
    int ffn_waves;     // wavefronts per bf16 FFN workgroup (1 or 4)
    int xcd_units;     // 1: each FFN work unit's workgroups on one XCD
    size_t esz, expert_bytes;
};

bool has_spatio(int mode) { return mode == CMOE_MODE_SPATIO_TEMPORAL || mode == CMOE_MODE_SPATIO_ONLY; }

cmoe_status validate(const cmoe_config* c, Derived* dv) {
    if (!c) return fail(CMOE_ERR_INVALID_ARG, "config is NULL");
    if (c->L < 1 || c->S < 1 || c->N < 1 || c->K < 1 || c->d < 1 || c->F < 1)
        return fail(CMOE_ERR_INVALID_ARG, "L, S, N, K, d and F must be >= 1");
    if (c->K > c->C) return fail(CMOE_ERR_INVALID_ARG, "capacity C must be at least K");
    if (c->C > c->N) return fail(CMOE_ERR_INVALID_ARG, "capacity C must not exceed N");
    if (c->mode != CMOE_MODE_TEMPORAL && c->mode != CMOE_MODE_SPATIO_TEMPORAL && c->mode != CMOE_MODE_SPATIO_ONLY)
        return fail(CMOE_ERR_INVALID_ARG, "unknown mode");
    if (c->policy < CMOE_POLICY_ROUTER || c->policy > CMOE_POLICY_LRFU)
        return fail(CMOE_ERR_INVALID_ARG, "unknown policy");
    if (c->mode == CMOE_MODE_SPATIO_ONLY && c->policy == CMOE_POLICY_ROUTER)
        return fail(CMOE_ERR_INVALID_ARG, "the Spatio-only mode has no Temporal Router: choose LRU, LFU or LRFU");
    if (c->mode == CMOE_MODE_SPATIO_TEMPORAL && c->policy != CMOE_POLICY_ROUTER)
        return fail(CMOE_ERR_UNSUPPORTED, "the full mode retains by the Temporal Router's s^T");
    if (c->policy == CMOE_POLICY_LRFU && !(std::isfinite(c->lrfu_lambda) && c->lrfu_lambda >= 0.0f))
        return fail(CMOE_ERR_INVALID_ARG, "lrfu_lambda must be finite and >= 0");
    if (c->R < 0 || c->R > c->N) return fail(CMOE_ERR_INVALID_ARG, "R must be in [0, N]");
    if (c->dtype != CMOE_F32 && c->dtype != CMOE_BF16) return fail(CMOE_ERR_INVALID_ARG, "unknown dtype");
    if (c->pool_kind != CMOE_POOL_DEVICE && c->pool_kind != CMOE_POOL_HOST_PINNED)
        return fail(CMOE_ERR_INVALID_ARG, "unknown pool kind");
    if (c->warmup_tokens < 0) return fail(CMOE_ERR_INVALID_ARG, "warmup_tokens must be >= 0");
    const int64_t max_slots = std::min<int64_t>(c->N, (int64_t)c->S * c->C);
    if (c->arena_slots < 0 || c->arena_slots > max_slots)
        return fail(CMOE_ERR_INVALID_ARG, "arena_slots must be in [0, min(N, S C)]");
    if (c->N > cmoe::kMaxN) return fail(CMOE_ERR_UNSUPPORTED, "N > 256 is not supported");
    if (c->K > cmoe::kMaxK) return fail(CMOE_ERR_UNSUPPORTED, "K > 64 is not supported");
    if (c->d % 64 || c->F % 64) return fail(CMOE_ERR_UNSUPPORTED, "d and F must be multiples of 64");
    if ((int64_t)c->S * c->K >= (int64_t)1 << 23) return fail(CMOE_ERR_UNSUPPORTED, "S*K too large");
    if ((c->flags & CMOE_FLAG_FFN_GROUPED) && (c->flags & CMOE_FLAG_FFN_SINGLE))
        return fail(CMOE_ERR_INVALID_ARG, "CMOE_FLAG_FFN_GROUPED and CMOE_FLAG_FFN_SINGLE exclude each other");
    if ((c->flags & CMOE_FLAG_FILL_ON_MAIN) && (c->flags & CMOE_FLAG_FILL_ON_SIDE))
        return fail(CMOE_ERR_INVALID_ARG, "CMOE_FLAG_FILL_ON_MAIN and CMOE_FLAG_FILL_ON_SIDE exclude each other");
    // grouped FFN workgroups pay off when buckets of more than 16 tokens are
    // common: by default, from 8 tokens per expert on average
    dv->ffn_waves = (c->flags & CMOE_FLAG_FFN_GROUPED) ? 4
                    : (c->flags & CMOE_FLAG_FFN_SINGLE) ? 1
                    : ((int64_t)c->S * c->K >= (int64_t)8 * c->N ? 4 : 1);
    // a work unit's workgroups on one XCD (its tokens' activations fetched
    // into one L2) pay off from 4 tokens per expert on average; with fewer,
    // spreading each unit over all XCDs streams the weights faster
    dv->xcd_units = (int64_t)c->S * c->K >= (int64_t)4 * c->N ? 1 : 0;
    dv->NW = (c->N + 63) / 64;
    const bool temporal = c->policy == CMOE_POLICY_ROUTER;
    dv->iT = temporal ? 1 : -1;
    dv->iS = has_spatio(c->mode) ? (temporal ? 2 : 1) : -1;
    dv->n_r = 1 + (temporal ? 1 : 0) + (has_spatio(c->mode) ? 1 : 0);
    dv->n_slots = c->arena_slots ? c->arena_slots : (int)max_slots;
    // the executed experts of a layer step (at most min(N, S K)) pass through a
    // smaller arena in rounds of n_slots
    const int64_t max_exec = std::min<int64_t>(c->N, (int64_t)c->S * c->K);
    dv->rounds = dv->n_slots < max_slots ? (int)((max_exec + dv->n_slots - 1) / dv->n_slots) : 1;
    dv->esz = c->dtype == CMOE_BF16 ? 2 : 4;
    dv->expert_bytes = (size_t)3 * c->d * c->F * dv->esz;
    // router split-K: each wavefront of a router workgroup sums a 32-aligned
    // k range of rdk; a workgroup covers kRouterWaves ranges and writes one
    // partial; at most kMaxSplit partials per logit, and ranges as long as
    // still give about a thousand wavefronts
    const int64_t tiles = (int64_t)dv->n_r * ((c->N + 15) / 16) * ((c->S + 15) / 16);
    const int W = cmoe::kRouterWaves;
    auto splits = [&](int64_t k) { return (c->d + W * k - 1) / (W * k); };
    int rdk = 32;
    while (splits(rdk) > cmoe::kMaxSplit) rdk *= 2;
    while (W * 2 * rdk <= c->d && tiles * W * splits(2 * rdk) >= 1024) rdk *= 2;
    // a single partial per logit leaves big layers (many streams, three
    // routers) with under two wavefronts per SIMD: take two
    if (splits(rdk) == 1 && tiles * W < 2048 && rdk >= 64) rdk /= 2;
    // up to four partials per logit (one slot group of the cache step's
    // loads) while the grid stays under ~8K wavefronts: shorter wavefronts
    // hide more of the loads' latency under the fp64 matrix work (measured on
    // MI355X, 256 streams with three routers: 11.3 against 12.2 us per launch
    // at d = 2048, 19.7 against 20.3 us at d = 4096)
    while (splits(rdk) < 4 && rdk >= 64 && splits(rdk / 2) <= 4 && tiles * W * splits(rdk / 2) <= 8192) rdk /= 2;
    dv->rdk = rdk;
    dv->nsplit = (int)splits(rdk);
    dv->zstride = dv->nsplit <= 4 ? 4 : cmoe::kMaxSplit;  // partial slots per logit
    return CMOE_OK;
}

// Offsets of every sub-buffer; used both for sizing and for carving.
struct Plan {
    size_t cache, aT, pol, pS, ctr, phys, active_sum, selcount, slot_of, slot_exp, slot_stamp, state_total;
    size_t zpart, logits, sel, gates, events, step_fills, bcount, pairs, act, yp, zero_row, units, round_of, ws_total;
    size_t arena;
};

int max_units(const cmoe_config* c) {
    return c->N + (int)(((int64_t)c->S * c->K + cmoe::kUnitTokens - 1) / cmoe::kUnitTokens);
}

Plan make_plan(const cmoe_config* c, const Derived& dv) {
    Plan p{};
    const size_t S = c->S, L = c->L, N = c->N, K = c->K;
    size_t o = 0;
    auto take = [&o](size_t bytes) {
        const size_t at = o;
        o += align256(bytes);
        return at;
    };
    p.cache = take(S * L * dv.NW * 8);
    p.aT = take(S * L * N * 4);
    p.pol = take(S * L * N * 4);
    p.pS = take(S * N * 4);
    p.ctr = take(S * L * cmoe::kNctr * 8);
    p.phys = take(L * 2 * 8);
    p.active_sum = take(L * 8);
    p.selcount = take(L * N * 8);
    p.slot_of = take(2 * L * N * 4);
    p.slot_exp = take(2 * L * (size_t)dv.n_slots * 4);
    p.slot_stamp = take(2 * L * (size_t)dv.n_slots * 4);
    p.state_total = o;
    o = 0;
    p.zpart = take(S * dv.n_r * N * (size_t)dv.zstride * 8);
    p.logits = take(L * S * dv.n_r * N * 4);
    p.sel = take(L * S * K * 4);
    p.gates = take(L * S * K * 4);
    p.events = take(L * S * 4 * 4);
    p.step_fills = take(L * 2 * 4);
    p.bcount = take(2 * N * 4);
    p.pairs = take(2 * N * S * 4);
    p.act = take(S * K * (size_t)c->F * dv.esz);
    p.yp = take(S * K * (size_t)c->d * dv.esz);
    p.zero_row = take(N * 4);
    p.units = take((size_t)max_units(c) * 16);
    p.round_of = take(N * 4);
    p.ws_total = o;
    p.arena = L * (size_t)dv.n_slots * dv.expert_bytes;
    return p;
}

// Points the workspace members of lo into the buffer wb (nullptr: none).
void bind_workspace(Layout& lo, char* wb, const Plan& p) {
    auto at = [wb](size_t off) -> char* { return wb ? wb + off : nullptr; };
    lo.zpart = reinterpret_cast<double*>(at(p.zpart));
    lo.logits = reinterpret_cast<float*>(at(p.logits));
    lo.sel = reinterpret_cast<int32_t*>(at(p.sel));
    lo.gates = reinterpret_cast<float*>(at(p.gates));
    lo.events = reinterpret_cast<int32_t*>(at(p.events));
    lo.step_fills = reinterpret_cast<int32_t*>(at(p.step_fills));
    lo.bcount = reinterpret_cast<int32_t*>(at(p.bcount));
    lo.pairs = reinterpret_cast<int32_t*>(at(p.pairs));
    lo.act = at(p.act);
    lo.yp = at(p.yp);
    lo.zero_row = reinterpret_cast<float*>(at(p.zero_row));
    lo.units = reinterpret_cast<int32_t*>(at(p.units));
    lo.round_of = reinterpret_cast<int32_t*>(at(p.round_of));
}

}  // namespace

struct cmoe_handle {
    cmoe_config cfg;
    Derived dv;
    Plan plan;
    Layout lo;                  // workspace pointers into the caller's workspace (null if none was given)
    Layout lo_static;           // the same with workspace pointers into the device's scratch array
    const Layout* cur = nullptr;  // the layout of the token being launched
    bool has_ws = false;        // the caller bound a workspace
    bool scratch_fits = false;  // the workspace plan fits the scratch array
    bool last_static = false;   // the last token ran on the scratch array
    int device = 0;
    hipStream_t main = nullptr, side = nullptr;
    bool side_is_main = true;
    std::vector<hipEvent_t> ev_access, ev_pro;
    int32_t t = 0;            // next token
    int64_t g = 0;            // layer steps accessed so far (bucket buffer parity)
    std::vector<int> ver;     // current slot-map version of each layer
    std::vector<int32_t> clk; // arena clock of each layer: advances once per fill launch
    int32_t R = 0;
    bool broken = false;
    // profiling
    int32_t prof_left = 0;
    uint32_t prof_mask = 0;
    std::vector<hipEvent_t> prof_pool;
    std::vector<std::pair<int, size_t>> prof_rec;  // kernel id, index of start event (stop = +1)
    size_t prof_next = 0;
};

namespace {

cmoe_status hip_fail(cmoe_handle* hd, hipError_t e, const char* where) {
    if (hd) hd->broken = true;
    return fail(CMOE_ERR_HIP, std::string("HIP error in ") + where + ": " + hipGetErrorString(e));
}

#define HIPCHK(expr, where)                                   \
    do {                                                      \
        hipError_t _e = (expr);                               \
        if (_e != hipSuccess) return hip_fail(hd, _e, where); \
    } while (0)

cmoe_status usable(cmoe_handle* hd) {
    if (!hd) return fail(CMOE_ERR_INVALID_ARG, "handle is NULL");
    if (hd->broken) return fail(CMOE_ERR_STATE, "handle unusable after an earlier HIP error; call cmoe_reset");
    return CMOE_OK;
}

// Runs launch(timing): when this kernel is being profiled, timing holds the
// next start/stop event pair, which the launch attaches to the kernel itself.
template <typename F>
hipError_t timed(cmoe_handle* hd, int kid, F&& launch) {
    cmoe::Timing tm;
    if (hd->prof_left > 0 && ((hd->prof_mask >> kid) & 1u) && hd->prof_next + 2 <= hd->prof_pool.size()) {
        const size_t i = hd->prof_next;
        hd->prof_next += 2;
        hd->prof_rec.emplace_back(kid, i);
        tm.start = hd->prof_pool[i];
        tm.stop = hd->prof_pool[i + 1];
    }
    return launch(tm);
}

// The arguments of one residency event of `layer` (or one FFN round of it);
// advances the layer's slot-map version and arena clock.
FillArgs event(cmoe_handle* hd, int layer, int kind, bool counted, bool zero_pre, int bbuf = 0, bool units = false,
               int round = 0) {
    FillArgs f{layer, kind, hd->ver[layer], counted ? 1 : 0, zero_pre ? 1 : 0, bbuf, units ? 1 : 0, round,
               ++hd->clk[layer]};
    hd->ver[layer] ^= 1;
    return f;
}

// One fill launch on stream st: event f, and event g of another layer if given.
hipError_t fill(cmoe_handle* hd, const FillArgs& f, hipStream_t st, const FillArgs* g = nullptr) {
    return timed(hd, KID_FILL, [&](const cmoe::Timing& tm) { return cmoe::launch_fill(*hd->cur, f, g, st, tm); });
}

// One decode token.  h == nullptr selects injected logits (no router, no FFN).
// on_scratch: the per-step buffers are the device's scratch array instead of
// the caller's workspace.
cmoe_status run_token(cmoe_handle* hd, const void* h, float* y, const float* zR, const float* zT, const float* zS,
                      bool on_scratch = false) {
    const cmoe_config& c = hd->cfg;
    hd->cur = on_scratch ? &hd->lo_static : &hd->lo;
    const Layout& lo = *hd->cur;
    const bool inject = h == nullptr;
    const bool refine_on = has_spatio(c.mode) && hd->t >= 1 && hd->R > 0;
    const bool counted = hd->t >= c.warmup_tokens;
    const uint32_t count = counted ? cmoe::kFlagCount : 0u;
    hipStream_t M = hd->main, Sd = hd->side;

    // A workspace that other calls used last may hold nonzero bucket counts:
    // the scratch array always (other handles share it), the caller's
    // workspace after tokens that ran on the scratch array.
    if (on_scratch || hd->last_static) HIPCHK(cmoe::launch_prep_workspace(lo, M), "workspace preparation");
    hd->last_static = on_scratch;

    if (refine_on) {  // layer 0: refined from the previous token's last-layer prediction
        StepArgs a{0, 0, hd->R, 0, cmoe::kFlagRefine | count, hd->t, {nullptr, nullptr, nullptr}};
        HIPCHK(timed(hd, KID_CACHE, [&](const cmoe::Timing& tm) { return cmoe::launch_cache_step(lo, a, M, tm); }),
               "refine layer 0");
        if (!hd->side_is_main) {
            HIPCHK(hipEventRecord(hd->ev_access[0], M), "event record");
            HIPCHK(hipStreamWaitEvent(Sd, hd->ev_access[0], 0), "stream wait");
        }
        HIPCHK(fill(hd, event(hd, 0, 1, counted, false), Sd), "fill");
        if (!hd->side_is_main) HIPCHK(hipEventRecord(hd->ev_pro[0], Sd), "event record");
    }
    for (int l = 0; l < c.L; ++l) {
        if (!inject)
            HIPCHK(timed(hd, KID_ROUTER, [&](const cmoe::Timing& tm) { return cmoe::launch_router(lo, l, h, M, tm); }),
                   "router");
        // the proactive fill of this layer reads its refined caches: it must end
        // before the access below changes them
        if (refine_on && !hd->side_is_main) HIPCHK(hipStreamWaitEvent(M, hd->ev_pro[l], 0), "stream wait");
        const bool refine_next = refine_on && l + 1 < c.L;
        uint32_t flags = cmoe::kFlagAccess | count;
        if (inject) flags |= cmoe::kFlagInject;
        if (refine_on) flags |= cmoe::kFlagRefinedHere;
        if (refine_next) flags |= cmoe::kFlagRefine;
        const int bbuf = (int)(hd->g & 1);
        StepArgs a{l, l + 1, hd->R, bbuf, flags, hd->t, {zR, nullptr, nullptr}};
        if (hd->dv.iT > 0) a.z[hd->dv.iT] = zT;
        if (hd->dv.iS > 0) a.z[hd->dv.iS] = zS;
        if (!inject && l > 0) {  // the same launch combines layer l - 1's expert outputs
            a.y = y;
            a.cl = l - 1;
        }
        HIPCHK(timed(hd, KID_CACHE, [&](const cmoe::Timing& tm) { return cmoe::launch_cache_step(lo, a, M, tm); }),
               "cache step");
        hd->g += 1;
        // Demand loads gate this layer's FFN; the same launch lays out the FFN
        // work units.  An arena smaller than the union of the caches runs the
        // FFN in rounds, each after the fill that brings its experts in.  The
        // proactive loads of layer l + 1 follow the same cache step: on the
        // main stream they join the first demand launch; on the side stream
        // they overlap this layer's FFN.
        for (int r = 0; r < hd->dv.rounds; ++r) {
            const FillArgs dem = event(hd, l, 0, counted, r == 0 && !refine_on, bbuf, !inject, r);
            if (r == 0 && refine_next && hd->side_is_main) {
                const FillArgs pro = event(hd, l + 1, 1, counted, false);
                HIPCHK(fill(hd, dem, M, &pro), "fill");
            } else {
                HIPCHK(fill(hd, dem, M), "fill");
            }
            if (r == 0 && refine_next && !hd->side_is_main) {
                HIPCHK(hipEventRecord(hd->ev_access[l], M), "event record");
                HIPCHK(hipStreamWaitEvent(Sd, hd->ev_access[l], 0), "stream wait");
                HIPCHK(fill(hd, event(hd, l + 1, 1, counted, false), Sd), "fill");
                HIPCHK(hipEventRecord(hd->ev_pro[l + 1], Sd), "event record");
            }
            if (!inject) {
                const int sv = hd->ver[l];
                HIPCHK(timed(hd, KID_UP,
                             [&](const cmoe::Timing& tm) {
                                 return cmoe::launch_ffn_up(lo, l, bbuf, sv, r, h, M, tm);
                             }),
                       "ffn up");
                HIPCHK(timed(hd, KID_DOWN,
                             [&](const cmoe::Timing& tm) { return cmoe::launch_ffn_down(lo, l, bbuf, sv, r, M, tm); }),
                       "ffn down");
            }
        }
    }
    if (!inject)
        HIPCHK(timed(hd, KID_COMBINE, [&](const cmoe::Timing& tm) { return cmoe::launch_combine(lo, c.L - 1, y, M, tm); }),
               "combine");
    hd->t += 1;
    if (hd->prof_left > 0) hd->prof_left -= 1;
    return CMOE_OK;
}

cmoe_status sync_all(cmoe_handle* hd) {
    HIPCHK(hipStreamSynchronize(hd->main), "stream synchronize");
    if (!hd->side_is_main) HIPCHK(hipStreamSynchronize(hd->side), "stream synchronize");
    return CMOE_OK;
}

}  // namespace

extern "C" {

cmoe_status cmoe_query(const cmoe_config* cfg, cmoe_sizes* out) {
    Derived dv;
    cmoe_status st = validate(cfg, &dv);
    if (st != CMOE_OK) return st;
    if (!out) return fail(CMOE_ERR_INVALID_ARG, "sizes output is NULL");
    const Plan p = make_plan(cfg, dv);
    out->arena_bytes = p.arena;
    out->state_bytes = p.state_total;
    out->workspace_bytes = p.ws_total;
    return CMOE_OK;
}

cmoe_status cmoe_init(const cmoe_config* cfg, const cmoe_weights* w, const cmoe_buffers* buf, void* main_stream,
                      void* side_stream, cmoe_handle** out) {
    if (out) *out = nullptr;
    Derived dv;
    cmoe_status st = validate(cfg, &dv);
    if (st != CMOE_OK) return st;
    if (!w || !buf || !out) return fail(CMOE_ERR_INVALID_ARG, "weights, buffers and output handle are required");
    if (!w->w_router || !w->cold_pool) return fail(CMOE_ERR_INVALID_ARG, "w_router and cold_pool are required");
    if (dv.iT > 0 && !w->w_temporal)
        return fail(CMOE_ERR_INVALID_ARG, "w_temporal is required with the router policy");
    if (dv.iS > 0 && !w->w_spatio)
        return fail(CMOE_ERR_INVALID_ARG, "w_spatio is required in the modes with a Spatio Router");
    if (!buf->arena || !buf->state) return fail(CMOE_ERR_INVALID_ARG, "arena and state buffers are required");
    for (const void* p : {buf->arena, buf->state, buf->workspace})
        if (reinterpret_cast<uintptr_t>(p) & 255) return fail(CMOE_ERR_INVALID_ARG, "buffers must be 256-byte aligned");
    const Plan plan = make_plan(cfg, dv);
    if (!buf->workspace && plan.ws_total > kScratchBytes)
        return fail(CMOE_ERR_UNSUPPORTED, "no workspace given and the per-step buffers (" +
                                              std::to_string(plan.ws_total) + " bytes) exceed the " +
                                              std::to_string(kScratchBytes) + "-byte scratch array");
    int device = 0;
    if (hipGetDevice(&device) != hipSuccess) {
        (void)hipGetLastError();
        return fail(CMOE_ERR_HIP, "hipGetDevice failed");
    }
    void* scratch_dev = nullptr;
    {
        const hipError_t e = scratch_on_device(device, &scratch_dev);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            return fail(CMOE_ERR_HIP, std::string("hipGetSymbolAddress of the scratch array: ") + hipGetErrorString(e));
        }
    }

    // The fill kernel reads the cold pool directly: resolve its device address
    // (a pinned host pool must be hipHostMalloc memory) and refuse pointers the
    // device cannot access rather than fault later.
    const void* pool_dev = w->cold_pool;
    if (cfg->pool_kind == CMOE_POOL_HOST_PINNED) {
        void* dptr = nullptr;
        if (hipHostGetDevicePointer(&dptr, const_cast<void*>(w->cold_pool), 0) != hipSuccess || !dptr) {
            (void)hipGetLastError();
            return fail(CMOE_ERR_INVALID_ARG, "cold_pool is not pinned, device-mapped host memory");
        }
        pool_dev = dptr;
    } else {
        hipPointerAttribute_t attr;
        if (hipPointerGetAttributes(&attr, w->cold_pool) != hipSuccess || attr.type != hipMemoryTypeDevice) {
            (void)hipGetLastError();
            return fail(CMOE_ERR_INVALID_ARG, "cold_pool is not device memory (use CMOE_POOL_HOST_PINNED for host)");
        }
    }

    cmoe_handle* hd = new cmoe_handle();
    hd->cfg = *cfg;
    hd->dv = dv;
    hd->plan = plan;
    hd->device = device;
    hd->has_ws = buf->workspace != nullptr;
    hd->scratch_fits = plan.ws_total <= kScratchBytes;
    hd->R = has_spatio(cfg->mode) ? cfg->R : 0;
    hd->ver.assign(cfg->L, 0);
    hd->clk.assign(cfg->L, 0);
    hd->main = static_cast<hipStream_t>(main_stream);
    // proactive loads run on the side stream only when asked for: joined to
    // the demand fill launch on the main stream they were faster on every
    // workload measured, a host pool included
    hd->side_is_main = side_stream == nullptr || side_stream == main_stream || !(cfg->flags & CMOE_FLAG_FILL_ON_SIDE);
    hd->side = hd->side_is_main ? hd->main : static_cast<hipStream_t>(side_stream);

    Layout& lo = hd->lo;
    const Plan& p = hd->plan;
    lo.L = cfg->L; lo.N = cfg->N; lo.K = cfg->K; lo.d = cfg->d; lo.F = cfg->F; lo.C = cfg->C; lo.S = cfg->S;
    lo.mode = cfg->mode; lo.dtype = cfg->dtype; lo.NW = dv.NW; lo.n_slots = dv.n_slots; lo.n_r = dv.n_r;
    lo.nsplit = dv.nsplit; lo.rdk = dv.rdk; lo.zstride = dv.zstride; lo.warmup = cfg->warmup_tokens;
    lo.iT = dv.iT; lo.iS = dv.iS; lo.policy = cfg->policy;
    lo.lrfu_w = (float)std::pow(2.0, -(double)cfg->lrfu_lambda);
    lo.expert_elems = (int64_t)3 * cfg->d * cfg->F;
    lo.rw[0] = w->w_router;
    lo.rw[1] = dv.iT == 1 ? w->w_temporal : (dv.iS == 1 ? w->w_spatio : nullptr);
    lo.rw[2] = dv.iS == 2 ? w->w_spatio : nullptr;
    lo.bias = w->logit_bias; lo.pool = pool_dev;
    lo.pool_host = cfg->pool_kind == CMOE_POOL_HOST_PINNED ? 1 : 0;
    lo.arena = buf->arena;
    char* sb = static_cast<char*>(buf->state);
    lo.cache = reinterpret_cast<unsigned long long*>(sb + p.cache);
    lo.aT = reinterpret_cast<float*>(sb + p.aT);
    lo.pol = reinterpret_cast<float*>(sb + p.pol);
    lo.pS = reinterpret_cast<float*>(sb + p.pS);
    lo.ctr = reinterpret_cast<int64_t*>(sb + p.ctr);
    lo.phys = reinterpret_cast<int64_t*>(sb + p.phys);
    lo.active_sum = reinterpret_cast<unsigned long long*>(sb + p.active_sum);
    lo.selcount = reinterpret_cast<unsigned long long*>(sb + p.selcount);
    lo.slot_of = reinterpret_cast<int32_t*>(sb + p.slot_of);
    lo.slot_exp = reinterpret_cast<int32_t*>(sb + p.slot_exp);
    lo.slot_stamp = reinterpret_cast<int32_t*>(sb + p.slot_stamp);
    lo.max_units = max_units(cfg);
    lo.ffn_waves = dv.ffn_waves;
    lo.xcd_units = dv.xcd_units;
    lo.unit_tokens = dv.ffn_waves > 1 ? cmoe::kUnitTokensGrouped : cmoe::kUnitTokens;
    hd->lo_static = lo;
    bind_workspace(lo, static_cast<char*>(buf->workspace), p);
    bind_workspace(hd->lo_static, hd->scratch_fits ? static_cast<char*>(scratch_dev) : nullptr, p);
    hd->cur = &hd->lo;

    auto mk = [&](hipEvent_t* e) { return hipEventCreateWithFlags(e, hipEventDisableTiming); };
    hd->ev_access.resize(cfg->L);
    hd->ev_pro.resize(cfg->L);
    hipError_t e = hipSuccess;
    for (int l = 0; l < cfg->L && e == hipSuccess; ++l) {
        e = mk(&hd->ev_access[l]);
        if (e == hipSuccess) e = mk(&hd->ev_pro[l]);
    }
    if (e == hipSuccess) e = cmoe::launch_init(lo, hd->main);
    if (e == hipSuccess) e = hipStreamSynchronize(hd->main);
    if (e != hipSuccess) {
        cmoe_destroy(hd);
        return fail(CMOE_ERR_HIP, std::string("HIP error in cmoe_init: ") + hipGetErrorString(e));
    }
    *out = hd;
    return CMOE_OK;
}

cmoe_status cmoe_step(cmoe_handle* hd, const void* h, float* y) {
    cmoe_status st = usable(hd);
    if (st != CMOE_OK) return st;
    if (!h || !y) return fail(CMOE_ERR_INVALID_ARG, "h and y are required");
    if (!hd->has_ws) return fail(CMOE_ERR_INVALID_ARG, "the handle has no workspace: use cmoe_step_noalloc");
    return run_token(hd, h, y, nullptr, nullptr, nullptr);
}

cmoe_status cmoe_step_noalloc(cmoe_handle* hd, const void* h, float* y) {
    cmoe_status st = usable(hd);
    if (st != CMOE_OK) return st;
    if (!h || !y) return fail(CMOE_ERR_INVALID_ARG, "h and y are required");
    if (!hd->scratch_fits)
        return fail(CMOE_ERR_UNSUPPORTED, "the per-step buffers (" + std::to_string(hd->plan.ws_total) +
                                              " bytes) exceed the " + std::to_string(kScratchBytes) +
                                              "-byte scratch array: use cmoe_step with a workspace");
    int device = -1;
    if (hipGetDevice(&device) != hipSuccess || device != hd->device) {
        (void)hipGetLastError();
        return fail(CMOE_ERR_INVALID_ARG, "the current device is not the one the handle was created on");
    }
    return run_token(hd, h, y, nullptr, nullptr, nullptr, true);
}

cmoe_status cmoe_step_logits(cmoe_handle* hd, const float* zR, const float* zT, const float* zS) {
    cmoe_status st = usable(hd);
    if (st != CMOE_OK) return st;
    if (!hd->has_ws) return fail(CMOE_ERR_INVALID_ARG, "the handle has no workspace: use cmoe_step_noalloc");
    if (!zR) return fail(CMOE_ERR_INVALID_ARG, "zR is required");
    if (hd->dv.iT > 0 && !zT) return fail(CMOE_ERR_INVALID_ARG, "zT is required with the router policy");
    if (hd->dv.iS > 0 && !zS) return fail(CMOE_ERR_INVALID_ARG, "zS is required in the modes with a Spatio Router");
    return run_token(hd, nullptr, nullptr, zR, zT, zS);
}

cmoe_status cmoe_stats(cmoe_handle* hd, cmoe_stats_t* total, int64_t* per_stream_layer, int64_t* per_layer_phys) {
    cmoe_status st = usable(hd);
    if (st != CMOE_OK) return st;
    st = sync_all(hd);
    if (st != CMOE_OK) return st;
    const cmoe_config& c = hd->cfg;
    std::vector<int64_t> ctr((size_t)c.S * c.L * cmoe::kNctr), phys((size_t)c.L * 2);
    HIPCHK(hipMemcpy(ctr.data(), hd->lo.ctr, ctr.size() * 8, hipMemcpyDeviceToHost), "counter read");
    HIPCHK(hipMemcpy(phys.data(), hd->lo.phys, phys.size() * 8, hipMemcpyDeviceToHost), "counter read");
    if (per_stream_layer) std::memcpy(per_stream_layer, ctr.data(), ctr.size() * 8);
    if (per_layer_phys) std::memcpy(per_layer_phys, phys.data(), phys.size() * 8);
    if (total) {
        cmoe_stats_t t{};
        for (int s = 0; s < c.S; ++s) {
            for (int l = 0; l < c.L; ++l) {
                const int64_t* v = &ctr[((size_t)s * c.L + l) * cmoe::kNctr];
                t.accesses += v[cmoe::kCtrA];
                t.hits += v[cmoe::kCtrHits];
                t.demand_misses += v[cmoe::kCtrD];
                t.proactive_loads += v[cmoe::kCtrP];
            }
            t.tokens += ctr[((size_t)s * c.L + 0) * cmoe::kNctr + cmoe::kCtrT];
        }
        for (int64_t v : phys) t.phys_fills += v;
        t.traffic_bytes = (t.demand_misses + t.proactive_loads) * (int64_t)hd->dv.expert_bytes;
        t.phys_bytes = t.phys_fills * (int64_t)hd->dv.expert_bytes;
        *total = t;
    }
    return CMOE_OK;
}

cmoe_status cmoe_get_cache(cmoe_handle* hd, int32_t stream, int32_t layer, int32_t* experts, int32_t* n) {
    cmoe_status st = usable(hd);
    if (st != CMOE_OK) return st;
    if (stream < 0 || stream >= hd->cfg.S || layer < 0 || layer >= hd->cfg.L || !experts || !n)
        return fail(CMOE_ERR_INVALID_ARG, "stream or layer out of range, or NULL output");
    st = sync_all(hd);
    if (st != CMOE_OK) return st;
    uint64_t w[4] = {0, 0, 0, 0};
    HIPCHK(hipMemcpy(w, hd->lo.cache + ((size_t)stream * hd->cfg.L + layer) * hd->dv.NW, hd->dv.NW * 8,
                     hipMemcpyDeviceToHost),
           "cache read");
    int k = 0;
    for (int e = 0; e < hd->cfg.N; ++e)
        if ((w[e >> 6] >> (e & 63)) & 1ull) {
            if (k < hd->cfg.C) experts[k] = e;
            ++k;
        }
    *n = k;
    return CMOE_OK;
}

cmoe_status cmoe_set_cache(cmoe_handle* hd, int32_t stream, int32_t layer, const int32_t* experts, int32_t n) {
    cmoe_status st = usable(hd);
    if (st != CMOE_OK) return st;
    if (stream < 0 || stream >= hd->cfg.S || layer < 0 || layer >= hd->cfg.L)
        return fail(CMOE_ERR_INVALID_ARG, "stream or layer out of range");
    if (n < 0 || n > hd->cfg.C || (n > 0 && !experts)) return fail(CMOE_ERR_INVALID_ARG, "need 0 <= n <= C experts");
    uint64_t w[4] = {0, 0, 0, 0};
    for (int i = 0; i < n; ++i) {
        const int e = experts[i];
        if (e < 0 || e >= hd->cfg.N) return fail(CMOE_ERR_INVALID_ARG, "expert index out of range");
        if ((w[e >> 6] >> (e & 63)) & 1ull) return fail(CMOE_ERR_INVALID_ARG, "duplicate expert");
        w[e >> 6] |= 1ull << (e & 63);
    }
    st = sync_all(hd);
    if (st != CMOE_OK) return st;
    HIPCHK(hipMemcpy(hd->lo.cache + ((size_t)stream * hd->cfg.L + layer) * hd->dv.NW, w, hd->dv.NW * 8,
                     hipMemcpyHostToDevice),
           "cache write");
    return CMOE_OK;
}

cmoe_status cmoe_set_R(cmoe_handle* hd, int32_t R) {
    cmoe_status st = usable(hd);
    if (st != CMOE_OK) return st;
    if (R < 0 || R > hd->cfg.N) return fail(CMOE_ERR_INVALID_ARG, "R must be in [0, N]");
    hd->R = has_spatio(hd->cfg.mode) ? R : 0;
    return CMOE_OK;
}

cmoe_status cmoe_reset(cmoe_handle* hd) {
    if (!hd) return fail(CMOE_ERR_INVALID_ARG, "handle is NULL");
    hd->broken = false;
    (void)hipGetLastError();
    cmoe_status st = sync_all(hd);
    if (st != CMOE_OK) return st;
    HIPCHK(cmoe::launch_init(hd->lo, hd->main), "reset");
    HIPCHK(hipStreamSynchronize(hd->main), "reset");
    hd->t = 0;
    hd->g = 0;
    hd->ver.assign(hd->cfg.L, 0);
    hd->clk.assign(hd->cfg.L, 0);
    return CMOE_OK;
}

cmoe_status cmoe_destroy(cmoe_handle* hd) {
    if (!hd) return CMOE_OK;
    if (hd->main) {
        (void)hipStreamSynchronize(hd->main);
        if (!hd->side_is_main) (void)hipStreamSynchronize(hd->side);
    }
    auto rm = [](hipEvent_t e) {
        if (e) (void)hipEventDestroy(e);
    };
    for (auto e : hd->ev_access) rm(e);
    for (auto e : hd->ev_pro) rm(e);
    for (auto e : hd->prof_pool) rm(e);
    delete hd;
    return CMOE_OK;
}

size_t cmoe_view_bytes(const cmoe_handle* hd, int32_t view) {
    if (!hd) return 0;
    const size_t S = hd->cfg.S, L = hd->cfg.L, N = hd->cfg.N, K = hd->cfg.K;
    switch (view) {
        case CMOE_VIEW_LOGITS: return L * S * hd->dv.n_r * N * 4;
        case CMOE_VIEW_SELECTED: return L * S * K * 4;
        case CMOE_VIEW_GATES: return L * S * K * 4;
        case CMOE_VIEW_CACHE: return S * L * hd->dv.NW * 8;
        case CMOE_VIEW_COUNTERS: return S * L * cmoe::kNctr * 8;
        case CMOE_VIEW_PHYS: return L * 2 * 8;
        case CMOE_VIEW_SLOTS: return L * N * 4;
        case CMOE_VIEW_EVENTS: return L * S * 4 * 4;
        case CMOE_VIEW_FILLS: return L * 2 * 4;
        case CMOE_VIEW_ACTIVE: return L * 8;
        case CMOE_VIEW_PRIORITY: return S * L * N * 4;
        case CMOE_VIEW_SELCOUNT: return L * N * 8;
        default: return 0;
    }
}

cmoe_status cmoe_read(cmoe_handle* hd, int32_t view, void* host_out, size_t bytes) {
    cmoe_status st = usable(hd);
    if (st != CMOE_OK) return st;
    const size_t need = cmoe_view_bytes(hd, view);
    if (need == 0) return fail(CMOE_ERR_INVALID_ARG, "unknown view");
    if (!host_out || bytes < need) return fail(CMOE_ERR_INVALID_ARG, "output buffer too small");
    // per-token outputs live where the last token ran
    const Layout& lo = (hd->last_static || !hd->has_ws) ? hd->lo_static : hd->lo;
    if (!lo.events) return fail(CMOE_ERR_STATE, "no per-step buffers to read");
    st = sync_all(hd);
    if (st != CMOE_OK) return st;
    if (view == CMOE_VIEW_SLOTS) {  // the current version of each layer's slot map
        const size_t N = hd->cfg.N;
        for (int l = 0; l < hd->cfg.L; ++l)
            HIPCHK(hipMemcpy(static_cast<char*>(host_out) + l * N * 4,
                             lo.slot_of + ((size_t)hd->ver[l] * hd->cfg.L + l) * N, N * 4, hipMemcpyDeviceToHost),
                   "view read");
        return CMOE_OK;
    }
    const void* src = nullptr;
    switch (view) {
        case CMOE_VIEW_LOGITS: src = lo.logits; break;
        case CMOE_VIEW_SELECTED: src = lo.sel; break;
        case CMOE_VIEW_GATES: src = lo.gates; break;
        case CMOE_VIEW_CACHE: src = lo.cache; break;
        case CMOE_VIEW_COUNTERS: src = lo.ctr; break;
        case CMOE_VIEW_PHYS: src = lo.phys; break;
        case CMOE_VIEW_EVENTS: src = lo.events; break;
        case CMOE_VIEW_FILLS: src = lo.step_fills; break;
        case CMOE_VIEW_ACTIVE: src = lo.active_sum; break;
        case CMOE_VIEW_PRIORITY: src = lo.pol; break;
        case CMOE_VIEW_SELCOUNT: src = lo.selcount; break;
    }
    HIPCHK(hipMemcpy(host_out, src, need, hipMemcpyDeviceToHost), "view read");
    return CMOE_OK;
}

cmoe_status cmoe_profile_begin(cmoe_handle* hd, int32_t max_tokens, uint32_t kernel_mask) {
    cmoe_status st = usable(hd);
    if (st != CMOE_OK) return st;
    if (max_tokens < 1) return fail(CMOE_ERR_INVALID_ARG, "max_tokens must be >= 1");
    hd->prof_mask = kernel_mask ? kernel_mask : ((1u << CMOE_KERNEL_COUNT) - 1u);
    int kinds = 0;
    for (int k = 0; k < CMOE_KERNEL_COUNT; ++k) kinds += (hd->prof_mask >> k) & 1u;
    const size_t per_token = ((size_t)hd->cfg.L * (hd->dv.rounds + 1) + 2) * kinds;  // timed launches per token, at most
    const size_t need = 2 * per_token * (size_t)max_tokens;
    while (hd->prof_pool.size() < need) {
        hipEvent_t e;
        HIPCHK(hipEventCreate(&e), "event create");
        hd->prof_pool.push_back(e);
    }
    hd->prof_rec.clear();
    hd->prof_next = 0;
    hd->prof_left = max_tokens;
    return CMOE_OK;
}

cmoe_status cmoe_profile_end(cmoe_handle* hd, double* ms_out, int64_t* launches_out) {
    cmoe_status st = usable(hd);
    if (st != CMOE_OK) return st;
    st = sync_all(hd);
    if (st != CMOE_OK) return st;
    std::vector<double> ms(CMOE_KERNEL_COUNT, 0.0);
    std::vector<int64_t> n(CMOE_KERNEL_COUNT, 0);
    for (const auto& r : hd->prof_rec) {
        float v = 0.0f;
        HIPCHK(hipEventElapsedTime(&v, hd->prof_pool[r.second], hd->prof_pool[r.second + 1]), "event elapsed");
        ms[r.first] += v;
        n[r.first] += 1;
    }
    if (ms_out) std::memcpy(ms_out, ms.data(), ms.size() * sizeof(double));
    if (launches_out) std::memcpy(launches_out, n.data(), n.size() * sizeof(int64_t));
    hd->prof_rec.clear();
    hd->prof_next = 0;
    hd->prof_left = 0;
    return CMOE_OK;
}

cmoe_status cmoe_concentration(cmoe_handle* hd, int32_t top_m, double* out4) {
    cmoe_status st = usable(hd);
    if (st != CMOE_OK) return st;
    if (!out4 || top_m < 1) return fail(CMOE_ERR_INVALID_ARG, "need top_m >= 1 and an output array");
    st = sync_all(hd);
    if (st != CMOE_OK) return st;
    const int L = hd->cfg.L, N = hd->cfg.N;
    std::vector<uint64_t> cnt((size_t)L * N);
    HIPCHK(hipMemcpy(cnt.data(), hd->lo.selcount, cnt.size() * 8, hipMemcpyDeviceToHost), "selection counts read");
    double acc[4] = {0.0, 0.0, 0.0, 0.0};
    int used = 0;
    std::vector<double> f(N);
    for (int l = 0; l < L; ++l) {
        const uint64_t* c = &cnt[(size_t)l * N];
        uint64_t tot = 0;
        for (int e = 0; e < N; ++e) tot += c[e];
        if (tot == 0) continue;
        double H = 0.0;
        for (int e = 0; e < N; ++e) {
            f[e] = (double)c[e] / (double)tot;
            if (f[e] > 0.0) H -= f[e] * std::log(f[e]);
        }
        std::vector<double> sorted(f);
        std::sort(sorted.begin(), sorted.end(), [](double a, double b) { return a > b; });
        double mass = 0.0;
        for (int i = 0; i < top_m && i < N; ++i) mass += sorted[i];
        acc[0] += std::exp(H);
        acc[1] += H;
        acc[2] += sorted[0];
        acc[3] += mass;
        ++used;
    }
    for (int i = 0; i < 4; ++i) out4[i] = used ? acc[i] / used : 0.0;
    return CMOE_OK;
}

cmoe_status cmoe_read_probe(const void* src, int64_t bytes, int32_t reps, double* gbps) {
    if (!src || !gbps) return fail(CMOE_ERR_INVALID_ARG, "read probe: src and gbps are required");
    if (reps < 1) return fail(CMOE_ERR_INVALID_ARG, "read probe: reps must be >= 1");
    if (bytes < ((int64_t)64 << 20)) return fail(CMOE_ERR_INVALID_ARG, "read probe: needs a buffer of at least 64 MiB");
    int64_t read = 0;
    const int64_t per_wave = cmoe::read_probe_units_per_wave(bytes, &read);
    cmoe_handle* hd = nullptr;  // no handle: errors do not mark one broken
    hipEvent_t e0 = nullptr, e1 = nullptr;
    hipError_t e = hipEventCreate(&e0);
    if (e == hipSuccess) e = hipEventCreate(&e1);
    float best = 0.0f;
    for (int32_t r = 0; e == hipSuccess && r < reps; ++r) {
        cmoe::Timing tm;
        tm.start = e0;
        tm.stop = e1;
        e = cmoe::launch_read_probe(src, per_wave, nullptr, tm);
        if (e == hipSuccess) e = hipEventSynchronize(e1);
        float ms = 0.0f;
        if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
        if (e == hipSuccess && (best == 0.0f || ms < best)) best = ms;
    }
    if (e1) (void)hipEventDestroy(e1);
    if (e0) (void)hipEventDestroy(e0);
    if (e != hipSuccess) return hip_fail(hd, e, "read probe");
    *gbps = (double)read / (best * 1e-3) / 1e9;
    return CMOE_OK;
}

const char* cmoe_last_error(void) { return g_err.c_str(); }

}  // extern "C"
