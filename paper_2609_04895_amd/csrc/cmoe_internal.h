// cmoe_internal.h - device layout and kernel launchers shared by the HIP
// translation units of libcmoe.so.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cmoe {

constexpr int kNctr = 5;          // per (stream, layer) counters: A, hits, D, P, T
constexpr int kCtrA = 0, kCtrHits = 1, kCtrD = 2, kCtrP = 3, kCtrT = 4;
constexpr int kMaxN = 256;        // experts per layer handled by the kernels
constexpr int kStreamsPerBlock = 4;   // cache-step kernel: one wavefront per stream

// Every pointer the kernels use, carved out of the caller's buffers.
struct Layout {
    int32_t L, N, K, d, F, C, S, mode, dtype, NW, n_slots, n_r, nsplit, rdk, n_tiles, warmup;
    int64_t expert_elems;  // 3 d F
    // weights
    const void* wR;
    const void* wT;
    const void* wS;
    const float* bias;
    const void* pool;
    // arena: [L][n_slots] experts
    void* arena;
    // state
    unsigned long long* cache;     // [S][L][NW]
    float* aT;           // [S][L][N]   s^T of the previous token (full mode)
    float* pS;           // [S][N]      latest Spatio Router distribution
    int64_t* ctr;        // [S][L][kNctr]
    int64_t* phys;       // [L][2]
    int64_t* active_sum; // [L]         distinct experts executed (counted tokens)
    int32_t* slot_of;    // [L][N]      slot of each expert, -1 absent
    int32_t* slot_exp;   // [L][n_slots] expert in each slot, -1 free
    uint32_t* tile_count; // [router tiles] splits finished per router tile
    // workspace
    double* zpart;       // [router tiles][nsplit][256] router partial sums
    float* logits;       // [L][S][n_r][N]
    int32_t* sel;        // [L][S][K]
    float* gates;        // [L][S][K]
    int32_t* events;     // [L][S][4]   hits, D, P, 0 of the last token
    int32_t* step_fills; // [L][2]
    int32_t* fill_list;  // [L][2][N][2] (expert, slot)
    int32_t* fill_count; // [L][2]
    unsigned long long* sel_mask;  // [S][NW] selected experts of the current layer
    int32_t* bcount;     // [N]         tokens per expert
    int32_t* boffset;    // [N]         first bucket position per expert
    int32_t* pairs;      // [S*K]       (stream << 8) | k, grouped by expert
    int32_t* active;     // [N]         experts with tokens, ascending
    int32_t* n_active;   // [1]
    void* act;           // [S*K][F]    SwiGLU intermediate (dtype)
    float* yp;           // [S][K][d]   gated expert outputs
};

// cache-step kernel flags
constexpr uint32_t kFlagAccess = 1u;       // route, access, retention for layer l
constexpr uint32_t kFlagInject = 2u;       // logits come from the caller
constexpr uint32_t kFlagRefine = 4u;       // refine layer `rl` (full mode)
constexpr uint32_t kFlagRefinedHere = 8u;  // layer l was refined earlier this token
constexpr uint32_t kFlagCount = 16u;       // this token is counted

struct StepArgs {
    int32_t l;          // layer accessed (kFlagAccess)
    int32_t rl;         // layer refined (kFlagRefine)
    int32_t R;          // refinement budget
    uint32_t flags;
    const float* zR;    // injected logits [S][L][N] (kFlagInject)
    const float* zT;
    const float* zS;
};

hipError_t launch_init(const Layout& lo, hipStream_t st);
hipError_t launch_router(const Layout& lo, int l, const void* h, hipStream_t st);
hipError_t launch_cache_step(const Layout& lo, const StepArgs& a, hipStream_t st);
hipError_t launch_finish(const Layout& lo, const StepArgs& a, hipStream_t st);
size_t finish_lds_bytes(const Layout& lo);  // dynamic LDS of the residency kernel
constexpr size_t kMaxFinishLds = 61440;
hipError_t launch_fill(const Layout& lo, int l, int kind, hipStream_t st);
hipError_t launch_ffn_up(const Layout& lo, int l, const void* h, hipStream_t st);
hipError_t launch_ffn_down(const Layout& lo, int l, hipStream_t st);
hipError_t launch_combine(const Layout& lo, int l, float* y, hipStream_t st);

}  // namespace cmoe
