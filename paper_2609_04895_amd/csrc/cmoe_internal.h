// cmoe_internal.h - device layout and kernel launchers shared by the HIP
// translation units of libcmoe.so.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cmoe {

constexpr int kNctr = 5;          // per (stream, layer) counters: A, hits, D, P, T
constexpr int kCtrA = 0, kCtrHits = 1, kCtrD = 2, kCtrP = 3, kCtrT = 4;
constexpr int kMaxN = 256;        // experts per layer handled by the kernels
constexpr int kMaxK = 64;         // Top-K handled by the kernels (one lane per selected expert)
constexpr int kMaxSplit = 16;        // router split-K partials per logit, at most
constexpr int kRouterWaves = 4;      // router: wavefronts per workgroup, one k sub-range each
constexpr int kStreamsPerBlock = 1;   // cache-step kernel: one wavefront per stream
// fill kernel workgroups: copies out of an HBM pool want many loads in
// flight (512 workgroups copy 2.7 times faster than 128); reads over the
// host link peak with fewer (128: 56 GB/s, 1024: 47 GB/s)
constexpr int kFillBlocksDevice = 512, kFillBlocksHost = 128;
// FFN work unit: one pass over an expert's weights for up to this many of its
// tokens: 64 with one wavefront per workgroup, 128 in the grouped launch
// (whose workgroups stage the activations in LDS for the four row tiles)
constexpr int kUnitTokens = 64, kUnitTokensGrouped = 128;

// Every pointer the kernels use, carved out of the caller's buffers.
struct Layout {
    int32_t L, N, K, d, F, C, S, mode, dtype, NW, n_slots, n_r, nsplit, rdk, zstride, warmup;
    int32_t iT, iS;        // router slot of the Temporal / Spatio Router, -1 if not used
    int32_t max_units;     // FFN work units per layer step, at most N + ceil(S K / kUnitTokens)
    int32_t unit_tokens;   // tokens per work unit: kUnitTokens, or kUnitTokensGrouped (grouped launch)
    int32_t ffn_waves;     // wavefronts per bf16 FFN workgroup: 1, or 4 (grouped: units of more
                           // than 16 tokens share their activations through LDS)
    int32_t xcd_units;     // 1: the bf16 FFN grids put each work unit's workgroups on one XCD,
                           // 0: on all XCDs in turn
    int32_t policy;        // retention priority (cmoe_policy)
    float lrfu_w;          // LRFU decay per token, fl32(2^-lambda)
    int64_t expert_elems;  // 3 d F
    // weights: router slot r (0 native, then temporal, then spatio, as used)
    const void* rw[3];
    const float* bias;
    const void* pool;
    int32_t pool_host;     // 1: the pool is pinned host memory read over the host link
    // arena: [L][n_slots] experts
    void* arena;
    // state
    unsigned long long* cache;  // [S][L][NW]  cache membership bits
    float* aT;                  // [S][L][N]   previous token's a-score: s^T (full mode),
                                //             p^R (Spatio-only mode)
    float* pol;                 // [S][L][N]   classical retention priority
    float* pS;                  // [S][N]      latest Spatio Router distribution
    int64_t* ctr;               // [S][L][kNctr]
    int64_t* phys;              // [L][2]      physical fills: demand, proactive
    unsigned long long* active_sum;  // [L]    distinct experts executed (counted tokens)
    unsigned long long* selcount;    // [L][N] native selections per expert (counted tokens)
    int32_t* slot_of;           // [2][L][N]   slot of each expert, -1 absent (two versions)
    int32_t* slot_exp;          // [2][L][n_slots] expert in each slot, -1 free
    int32_t* slot_stamp;        // [2][L][n_slots] arena clock at the last use of each slot's expert
    // workspace
    double* zpart;              // [S][n_r][N][zstride] router partial sums
    float* logits;              // [L][S][n_r][N]
    int32_t* sel;               // [L][S][K]
    float* gates;               // [L][S][K]
    int32_t* events;            // [L][S][4]   hits, D, P, 0 of the last token
    int32_t* step_fills;        // [L][2]      physical fills of the last token
    int32_t* bcount;            // [2][N]      tokens per expert (two buffers)
    int32_t* pairs;             // [2][N][S]   (stream << 8) | k of each token of an expert
    void* act;                  // [S][K][F]   SwiGLU intermediate (dtype)
    void* yp;                   // [S][K][d]   gated expert outputs (dtype)
    float* zero_row;            // [N]         zeros (native bias when there is none)
    int32_t* units;             // [max_units][4] FFN work units of the current round, heaviest
                                //             first: {(pass << 8) | expert, slot, tokens, 0},
                                //             {-1, -1, 0, 0} past the end
    int32_t* round_of;          // [N]         FFN round of each expert executed by the layer
                                //             step, -1 if not executed
};

// cache-step kernel flags
constexpr uint32_t kFlagAccess = 1u;       // route, access, retention for layer l
constexpr uint32_t kFlagInject = 2u;       // logits come from the caller
constexpr uint32_t kFlagRefine = 4u;       // refine layer `rl` (modes with a Spatio Router)
constexpr uint32_t kFlagRefinedHere = 8u;  // layer l was refined earlier this token
constexpr uint32_t kFlagCount = 16u;       // this token is counted

struct StepArgs {
    int32_t l;          // layer accessed (kFlagAccess)
    int32_t rl;         // layer refined (kFlagRefine)
    int32_t R;          // refinement budget
    int32_t bbuf;       // bucket buffer of this layer step (the other one is cleared)
    uint32_t flags;
    int32_t t;          // token index (LRU clock)
    const float* z[3];  // injected logits [S][L][N] per router slot (kFlagInject)
    float* y;           // non-NULL: the launch also combines layer cl's expert outputs into y
    int32_t cl;
};

// One residency event of layer `layer` (or one round of it): the arena must
// hold the union of the streams' caches, or, when the union does not fit,
// the experts of this FFN round.  Slot maps and stamps are read from version
// rv and written to version rv ^ 1.
struct FillArgs {
    int32_t layer;
    int32_t kind;        // 0 after the post-access update, 1 after refinement
    int32_t rv;
    int32_t counted;
    int32_t zero_pre;    // kind 0: no refinement happened this token, clear its fill count
    int32_t bbuf;        // kind 0: bucket buffer of the layer step (its counts give the executed experts)
    int32_t units;       // kind 0: lay out the FFN work units of this round
    int32_t round;       // kind 0: FFN round of the layer step (0 plans the rounds)
    int32_t clk;         // arena clock of this launch: the last use it stamps
};

// Optional timing of one launch: with events, they take the kernel's own
// start and end timestamps (hipExtLaunchKernel), not those of markers
// recorded on the stream around the launch.
struct Timing {
    hipEvent_t start = nullptr, stop = nullptr;
};

template <typename... KArgs, typename... Args>
inline void launch_kernel(void (*kernel)(KArgs...), dim3 grid, dim3 block, hipStream_t st, const Timing& tm,
                          Args... args) {
    if (tm.start)
        hipExtLaunchKernelGGL(kernel, grid, block, 0, st, tm.start, tm.stop, 0, args...);
    else
        hipLaunchKernelGGL(kernel, grid, block, 0, st, args...);
}

hipError_t launch_init(const Layout& lo, hipStream_t st);  // state, and the workspace if bound
hipError_t launch_prep_workspace(const Layout& lo, hipStream_t st);
hipError_t launch_router(const Layout& lo, int l, const void* h, hipStream_t st, const Timing& tm = {});
hipError_t launch_cache_step(const Layout& lo, const StepArgs& a, hipStream_t st, const Timing& tm = {});
// g (or NULL): a second event of another layer in the same launch
hipError_t launch_fill(const Layout& lo, const FillArgs& f, const FillArgs* g, hipStream_t st,
                       const Timing& tm = {});
hipError_t launch_ffn_up(const Layout& lo, int l, int bbuf, int sv, int round, const void* h, hipStream_t st,
                         const Timing& tm = {});
hipError_t launch_ffn_down(const Layout& lo, int l, int bbuf, int sv, int round, hipStream_t st,
                           const Timing& tm = {});
hipError_t launch_combine(const Layout& lo, int l, float* y, hipStream_t st, const Timing& tm = {});
// streaming read of per_wave 16-byte units by each wavefront of the probe
// grid; read_probe_units_per_wave gives the largest per_wave that fits in
// `bytes` and the bytes the grid then reads
int64_t read_probe_units_per_wave(int64_t bytes, int64_t* read_bytes);
hipError_t launch_read_probe(const void* src, int64_t per_wave, hipStream_t st, const Timing& tm);

}  // namespace cmoe
