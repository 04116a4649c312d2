/*
 * cmoe.h - C ABI of the cache-aware MoE decode step on one MI355X (gfx950).
 *
 * The library runs, for S independent decode streams and L MoE layers in
 * causal order, one decode token per call:
 *   - the native router p^R = softmax(W^R h), S_t = TopK(p^R)            (Section 2)
 *   - the Temporal Router p^T = softmax(W^T h), s^T = p^R + p^T         (Section 3.2)
 *   - in full mode the Spatio Router p^S = softmax(W^S h) of the causal
 *     predecessor and the pre-access refinement over Top_R(a^T + p^S)    (Section 3.3,
 *                                                                         Algorithm 2)
 *   - the post-access retention update U_C of each per-(stream, layer)
 *     cache of capacity C                                                (Algorithm 1)
 *     with the Temporal Router's s^T as priority, or one of the classical
 *     cache-update baselines LRU, LFU, LRFU                              (Section 4.1,
 *                                                                         Table 1)
 *   - the Spatio-only ablation: refinement over Top_R(p^R_{t-1} + p^S)
 *     with classical eviction of demand misses                           (Section 5,
 *                                                                         Appendix B.4)
 *   - the accounting of accesses A, hits, demand misses D, proactive
 *     loads P, decode tokens T and expert-weight traffic (D + P) S_exp    (Section 4.1)
 *   - copies of newly needed experts from a cold pool into HBM slots
 *     (a side HIP stream), and the SwiGLU expert FFN on the resident
 *     weights ("execute the MoE layer", Algorithm 2).
 * Notation follows the paper's problem statement (Section 2): L layers, N
 * experts per layer, native Top-K, per-layer cache capacity C (the paper's
 * B, with C >= K), refinement budget R (Appendix B.2, "replace_lowest").
 *
 * Conventions for every entry point:
 *   - returns a cmoe_status; nothing throws, aborts or prints;
 *   - on failure cmoe_last_error() describes the cause (thread-local string,
 *     valid until the next call on the same thread);
 *   - device pointers are HIP device addresses (or host-pinned addresses
 *     where stated); the caller allocates and owns every buffer and both
 *     streams, which must outlive the handle; the library calls no hipMalloc;
 *   - a HIP failure is sticky: the call returns CMOE_ERR_HIP and later calls
 *     on the handle return CMOE_ERR_STATE until cmoe_reset or cmoe_destroy;
 *   - a handle is used by one host thread at a time.
 */
#ifndef CMOE_H
#define CMOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    CMOE_OK = 0,
    CMOE_ERR_INVALID_ARG = -1, /* a value violates the problem statement       */
    CMOE_ERR_UNSUPPORTED = -2, /* valid, but outside what the kernels handle   */
    CMOE_ERR_HIP = -3,         /* the HIP runtime reported an error            */
    CMOE_ERR_STATE = -4        /* handle unusable after an earlier HIP error   */
} cmoe_status;

typedef enum {
    CMOE_MODE_TEMPORAL = 0,         /* update-only: no refinement (Section 3.2)    */
    CMOE_MODE_SPATIO_TEMPORAL = 1,  /* full mode with refinement (Section 3.3)     */
    CMOE_MODE_SPATIO_ONLY = 2       /* refinement by p^R_{t-1} + p^S, classical
                                       retention (Section 5, Appendix B.4)         */
} cmoe_mode;

/* Retention priority of the post-access update (Algorithm 1): the selected
 * experts are protected and, when the cache is full, each demand-loaded
 * expert replaces the lowest-priority resident that is not selected now
 * (lower expert index on ties).  The classical priorities follow their
 * textbook definitions and are updated at every access before the eviction:
 *   LRU   time of the last use (two events per token t: refinement at 2t + 1,
 *         access at 2t + 2; a proactively inserted expert takes 2t + 1);
 *   LFU   number of selections;
 *   LRFU  C <- fl32(C * w) (+ 1 if selected) for every expert,
 *         w = fl32(2^-lrfu_lambda) (Lee et al. 2001).
 * They use the native router only.  CMOE_MODE_SPATIO_TEMPORAL needs
 * CMOE_POLICY_ROUTER; CMOE_MODE_SPATIO_ONLY needs a classical policy. */
typedef enum {
    CMOE_POLICY_ROUTER = 0,  /* s^T = p^R + p^T of the Temporal Router           */
    CMOE_POLICY_LRU = 1,
    CMOE_POLICY_LFU = 2,
    CMOE_POLICY_LRFU = 3
} cmoe_policy;

typedef enum {
    CMOE_F32 = 0,  /* fp32 weights and hidden states                          */
    CMOE_BF16 = 1  /* bf16 weights and hidden states, fp32 accumulation        */
} cmoe_dtype;

typedef enum {
    CMOE_POOL_DEVICE = 0,      /* cold pool in device memory                  */
    CMOE_POOL_HOST_PINNED = 1  /* cold pool in pinned, device-mapped host RAM  */
} cmoe_pool_kind;

/* flags.  Demand fills always run on the main stream: they gate the layer's
 * FFN.  The proactive fills of layer l + 1 follow layer l's cache step: by
 * default they join layer l's demand fill launch on the main stream; with
 * CMOE_FLAG_FILL_ON_SIDE (and a side stream) they run on the side stream,
 * overlapping layer l's FFN.  Both flags: CMOE_ERR_INVALID_ARG. */
#define CMOE_FLAG_FILL_ON_MAIN 0x1u /* proactive fills on the main stream (the default)      */
#define CMOE_FLAG_FILL_ON_SIDE 0x8u /* proactive fills on the side stream                    */
/* bf16 expert FFN launch shape.  Single: one wavefront per workgroup, each on
 * its own row tile.  Grouped: four wavefronts per workgroup on consecutive row
 * tiles of one work unit; units of more than 16 tokens load their activations
 * once per workgroup into LDS.  Default: grouped when S K >= 8 N (at least 8
 * tokens per expert on average), else single.  Both flags: CMOE_ERR_INVALID_ARG.
 * The results are the same either way. */
#define CMOE_FLAG_FFN_GROUPED 0x2u
#define CMOE_FLAG_FFN_SINGLE 0x4u

/* Problem shape.  Valid values: 1 <= K <= C <= N (Section 2: capacity at least
 * Top-K); 0 <= R <= N; L, S >= 1; d, F >= 1; warmup_tokens >= 0; a known mode
 * and policy, paired as cmoe_policy states; lrfu_lambda finite and >= 0 with
 * CMOE_POLICY_LRFU; 0 <= arena_slots <= min(N, S C).  Supported: N <= 256, d
 * and F multiples of 64.  R is ignored in CMOE_MODE_TEMPORAL.
 *
 * Physical residency.  Each layer's HBM arena has arena_slots expert slots
 * (0: min(N, S C), which always holds the union of the streams' caches).
 * While the union of the caches fits, the arena holds all of it: an expert
 * that leaves every cache frees its slot, a new one takes the lowest free slot
 * (ascending expert order), after refinement and after the post-access update.
 * When it does not fit (the paper's bounded device cache, Section 3.1 and the
 * Figure 1 caption, with more streams than slots), the arena is a second-level
 * cache: the layer step's FFN runs in rounds of at most arena_slots of the
 * experts it executes (those already resident first, then the others, each
 * group in ascending order); a missing expert takes the lowest free slot or
 * evicts the least recently used expert that no remaining round needs (lower
 * slot on equal recency); after refinement only free slots are filled. */
typedef struct {
    int32_t L, N, K, d, F, C, R, S;
    int32_t mode;          /* cmoe_mode                                         */
    int32_t dtype;         /* cmoe_dtype of weights and hidden states           */
    int32_t pool_kind;     /* cmoe_pool_kind                                    */
    int32_t warmup_tokens; /* leading tokens whose transfers are not counted
                              (the paper excludes prefill transfers)            */
    uint32_t flags;
    int32_t policy;        /* cmoe_policy                                       */
    float lrfu_lambda;     /* LRFU recency weight (the paper uses 0.5)          */
    int32_t arena_slots;   /* HBM expert slots per layer; 0: min(N, S C)        */
} cmoe_config;

/* Weights (device pointers unless stated).  Router matrices are bias-free
 * d -> N maps per layer, row-major [L][N][d] in the config dtype.  The cold
 * pool holds every expert, [L][N] x expert_bytes, each expert laid out as
 * W_gate[F][d], W_up[F][d], W_down[d][F]; expert_bytes = 3 d F sizeof(dtype).
 * With CMOE_POOL_HOST_PINNED, cold_pool is a pinned host address mapped into
 * the device (hipHostMalloc). */
typedef struct {
    const void* w_router;    /* W^R [L][N][d]                                    */
    const void* w_temporal;  /* W^T [L][N][d]; required with CMOE_POLICY_ROUTER,
                                else ignored                                     */
    const void* w_spatio;    /* W^S [L][N][d]; required in the two modes with a
                                Spatio Router, else ignored                      */
    const float* logit_bias; /* [L][N] fp32 added to native logits, or NULL      */
    const void* cold_pool;   /* [L][N][expert_bytes]                             */
} cmoe_weights;

/* Device buffer sizes in bytes; every buffer must be 256-byte aligned. */
typedef struct {
    size_t arena_bytes;     /* HBM expert slots: L x arena_slots experts         */
    size_t state_bytes;     /* caches, scores, counters, slot maps               */
    size_t workspace_bytes; /* per-step scratch and the inspectable outputs      */
} cmoe_sizes;

typedef struct {
    void* arena;
    void* state;
    void* workspace;
} cmoe_buffers;

/* Totals over all streams and layers, counted tokens only.  traffic_bytes =
 * (demand_misses + proactive_loads) x expert_bytes (Section 4.1 "Metrics");
 * phys_fills counts expert copies into the HBM slots, phys_bytes their bytes. */
typedef struct {
    int64_t accesses, hits, demand_misses, proactive_loads, tokens, traffic_bytes;
    int64_t phys_fills, phys_bytes;
} cmoe_stats_t;

typedef struct cmoe_handle cmoe_handle;

/* Buffer sizes for a configuration.  Validates it as cmoe_init does.  Pure host
 * code: needs no GPU. */
cmoe_status cmoe_query(const cmoe_config* cfg, cmoe_sizes* out);

/* Binds weights and buffers, clears the state (empty caches, zero counters, no
 * resident experts) on main_stream and returns a handle.  side_stream may be
 * NULL (then fills run on main_stream).  Streams are hipStream_t values.
 * buf->workspace may be NULL for a handle that runs every token through
 * cmoe_step_noalloc; its per-step buffers must then fit the scratch array
 * (CMOE_ERR_UNSUPPORTED otherwise).  The handle belongs to the device that is
 * current during this call. */
cmoe_status cmoe_init(const cmoe_config* cfg, const cmoe_weights* w, const cmoe_buffers* buf,
                      void* main_stream, void* side_stream, cmoe_handle** out);

/* One decode token for all streams, asynchronous on main_stream.
 * h: [S][L][d] hidden states h_{t,l} in the config dtype (device).
 * y: [S][L][d] fp32 output of each MoE layer (device), valid once main_stream
 *    has completed.  The token index t is kept by the handle. */
cmoe_status cmoe_step(cmoe_handle* hd, const void* h, float* y);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): cmoe_step
 * with the per-step buffers (router partials, logits, selections, gates,
 * buckets, work units, the SwiGLU intermediate and the gated expert outputs)
 * in a scratch array that the library holds on each device, 64 MiB, instead
 * of the handle's workspace.  Allocates nothing; the same kernels, inputs,
 * outputs and results as cmoe_step.  Every call on a device shares that
 * device's array and leaves its contents behind (each call clears what must
 * start at zero); calls that overlap in time on one device race, so calls of
 * different handles must be ordered (one stream, or synchronized).  The views
 * of per-token outputs then read the scratch array until the next cmoe_step.
 * CMOE_ERR_UNSUPPORTED when the configuration's per-step buffers exceed
 * 64 MiB; CMOE_ERR_INVALID_ARG when the current device is not the handle's. */
cmoe_status cmoe_step_noalloc(cmoe_handle* hd, const void* h, float* y);

/* The cache path of one token from given fp32 logits, without the router
 * GEMV and without the FFN: softmax, Top-K, refinement, access, retention,
 * counters, residency and fills.  zR (native, bias already added), zT, zS:
 * [S][L][N] fp32 (device); zT is required with CMOE_POLICY_ROUTER and zS in
 * the modes with a Spatio Router; otherwise they are ignored (may be NULL). */
cmoe_status cmoe_step_logits(cmoe_handle* hd, const float* zR, const float* zT, const float* zS);

/* Synchronizes both streams and reads the counters.  total may be NULL.
 * per_stream_layer (or NULL): [S][L][5] int64 = A, hits, D, P, T.
 * per_layer_phys (or NULL): [L][2] int64 = demand fills, proactive fills. */
cmoe_status cmoe_stats(cmoe_handle* hd, cmoe_stats_t* total, int64_t* per_stream_layer,
                       int64_t* per_layer_phys);

/* Reads the cache C of (stream, layer): its experts in ascending order into
 * experts[0..n) (experts must hold C entries).  Synchronizes. */
cmoe_status cmoe_get_cache(cmoe_handle* hd, int32_t stream, int32_t layer, int32_t* experts,
                           int32_t* n);

/* Replaces the cache of (stream, layer) with n <= C distinct experts.  Only the
 * logical cache changes; physical residency follows at that layer's next
 * residency event.  Synchronizes. */
cmoe_status cmoe_set_cache(cmoe_handle* hd, int32_t stream, int32_t layer, const int32_t* experts,
                           int32_t n);

/* Changes the refinement budget R (0 <= R <= N) for the following tokens; an
 * inference-time knob that needs no retraining (Section 3.3). */
cmoe_status cmoe_set_R(cmoe_handle* hd, int32_t R);

/* Empty caches, zero counters and scores, no resident experts, t = 0.  Also
 * clears a sticky HIP error. */
cmoe_status cmoe_reset(cmoe_handle* hd);

/* Releases the handle (not the caller's buffers).  NULL is accepted. */
cmoe_status cmoe_destroy(cmoe_handle* hd);

/* Inspectable state (all synchronize).  Layouts:
 *   CMOE_VIEW_LOGITS    fp32  [L][S][n_r][N] logits used by the last token:
 *                              native, then temporal (router policy), then
 *                              spatio (modes with a Spatio Router)
 *   CMOE_VIEW_SELECTED  int32 [L][S][K] selected experts, descending logit
 *   CMOE_VIEW_GATES     fp32  [L][S][K] renormalised selected probabilities
 *   CMOE_VIEW_CACHE     u64   [S][L][W] cache membership bit masks,
 *                              W = ceil(N / 64), expert e is bit e % 64 of word e / 64
 *   CMOE_VIEW_COUNTERS  int64 [S][L][5] A, hits, D, P, T
 *   CMOE_VIEW_PHYS      int64 [L][2] physical fills: demand, proactive
 *   CMOE_VIEW_SLOTS     int32 [L][N] HBM slot of each expert, -1 if absent
 *   CMOE_VIEW_EVENTS    int32 [L][S][4] last token: hits, D, P, 0
 *   CMOE_VIEW_FILLS     int32 [L][2] last token's physical fills: demand, proactive
 *   CMOE_VIEW_ACTIVE    int64 [L] distinct experts executed by the FFN, summed
 *                              over counted tokens (each is one read of its weights)
 *   CMOE_VIEW_PRIORITY  fp32  [S][L][N] classical retention priority (LRU time,
 *                              LFU count, LRFU value); zeros with the router policy
 *   CMOE_VIEW_SELCOUNT  u64   [L][N] native selections of each expert, summed over
 *                              streams and counted tokens */
enum {
    CMOE_VIEW_LOGITS = 0,
    CMOE_VIEW_SELECTED = 1,
    CMOE_VIEW_GATES = 2,
    CMOE_VIEW_CACHE = 3,
    CMOE_VIEW_COUNTERS = 4,
    CMOE_VIEW_PHYS = 5,
    CMOE_VIEW_SLOTS = 6,
    CMOE_VIEW_EVENTS = 7,
    CMOE_VIEW_FILLS = 8,
    CMOE_VIEW_ACTIVE = 9,
    CMOE_VIEW_PRIORITY = 10,
    CMOE_VIEW_SELCOUNT = 11,
    CMOE_VIEW_COUNT = 12
};

/* Bytes of a view (0 for an unknown view or a NULL handle). */
size_t cmoe_view_bytes(const cmoe_handle* hd, int32_t view);

/* Copies a view into host memory of at least cmoe_view_bytes bytes. */
cmoe_status cmoe_read(cmoe_handle* hd, int32_t view, void* host_out, size_t bytes);

/* Per-kernel timing with HIP events.  cmoe_profile_begin makes the next
 * max_tokens calls of cmoe_step / cmoe_step_logits attach a start/stop event
 * pair to each launch of the kernels selected by kernel_mask (bit i = kernel
 * id i; 0 selects all): the events take the kernel's own start and end
 * timestamps (hipExtLaunchKernel);
 * cmoe_profile_end synchronizes and returns, per kernel id, the summed
 * milliseconds and the launch count.  Kernel ids: 0 router GEMV, 1 cache
 * step (routing, refinement, retention, counters, expert grouping; from the
 * second layer on, the same launch also runs the previous layer's combine),
 * 2 residency and fill, 3 expert gate/up, 4 expert down, 5 combine of the
 * last layer (one launch per token).
 * ms_out and launches_out hold CMOE_KERNEL_COUNT entries.  Timed launches
 * carry extra bookkeeping; time few kernels at once. */
#define CMOE_KERNEL_COUNT 6
cmoe_status cmoe_profile_begin(cmoe_handle* hd, int32_t max_tokens, uint32_t kernel_mask);
cmoe_status cmoe_profile_end(cmoe_handle* hd, double* ms_out, int64_t* launches_out);

/* Expert-use concentration of the native selections so far (Section 5,
 * routing behaviour): per layer with at least one counted selection, the
 * selection frequencies f_e (summing to 1), entropy H = -sum f_e ln f_e;
 * out4 = the means over those layers of {exp(H) (effective experts), H,
 * max_e f_e, the sum of the top_m largest f_e} (the paper uses top_m = 8).
 * All zeros before any counted token.  Synchronizes. */
cmoe_status cmoe_concentration(cmoe_handle* hd, int32_t top_m, double* out4);

/* Measurement utility, not part of the decode path: the rate at which the
 * current device streams `bytes` of device memory at src with the access
 * pattern of the expert weight loads (16-byte nontemporal loads, one
 * contiguous kilobyte per wavefront instruction, eight in flight, each
 * wavefront walking its own contiguous block).  It is the practical ceiling of
 * the FFN's weight stream, as opposed to the datasheet peak.  src: device
 * memory owned by the caller, only read (its contents do not matter);
 * bytes >= 64 MiB (a smaller buffer cannot occupy the device); the part read
 * is the largest multiple of the probe's block size that fits.  Runs `reps`
 * >= 1 launches on the null stream of the current device, synchronizes, and
 * writes the best rate in GB/s (10^9 bytes per second) to *gbps.  Allocates
 * nothing. */
cmoe_status cmoe_read_probe(const void* src, int64_t bytes, int32_t reps, double* gbps);

const char* cmoe_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* CMOE_H */
