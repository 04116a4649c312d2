// ffn.hip - the SwiGLU expert FFN over the resident expert weights
// ("execute the MoE layer", Algorithm 2), grouped by expert:
//   a_e = silu(W_gate,e x) * (W_up,e x),  y_(s,k) = g_(s,k) W_down,e a_e,
//   y_s = sum_k y_(s,k)  (k in ascending order).
// Each expert's weights are read from its HBM slot once per work unit (a
// pass over up to 64 of its tokens; nearly every expert needs one), so the
// layer step streams about |union of selected experts| x expert_bytes: the
// kernels are HBM-bound.
//
// bf16: one wavefront per 16 rows of W_gate and of W_up (gate/up kernel) or
// per 32 rows of W_down (down kernel), one wavefront per workgroup or four
// (grouped: consecutive row tiles of one unit, big units sharing their
// activations through LDS), on the bf16 matrix core
// (v_mfma_f32_16x16x32_bf16, fp32 accumulation).  The expert's tokens form the
// 16 columns of the B operand (groups of 16 tokens; several groups reuse the
// loaded weights).  Per 64-wide k chunk, lane (r, g) of the A operand holds
// W[row r][kc + 8 g .. + 8] and W[row r][kc + 32 + 8 g .. + 8]; the two MFMAs
// of a chunk take k-slots kc + 8 g + {0..7} and kc + 32 + 8 g + {0..7}, the
// same for both operands.  Each activation load thus reads one contiguous
// 64-byte half of a token's 128-byte k chunk.
// The weights come from the expert's HBM slot in packed order (the fill
// kernel writes it so): each A operand load of a wavefront reads one
// contiguous kilobyte and each wavefront streams one contiguous block.  The
// SwiGLU intermediate is stored in bf16 (the input type of the down kernel's
// matrix core).
//
// fp32: VALU kernels, one lane per output row, fp32 accumulation, over
// transposed weights (the fill kernel writes them so): the lanes of a
// wavefront read consecutive floats for each k, 32 k at a time.
#include "cmoe_internal.h"

namespace cmoe {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kNG = 4;          // token groups (of 16) per pass when a unit holds more than 16
static_assert(kUnitTokens == 16 * kNG, "one work unit is one pass over the weights");
constexpr int kUnroll = 4;      // k chunks per load block, one token group
constexpr int kUnrollWide = 2;  // k chunks per load block, kNG token groups sharing LDS (grouped launch)
constexpr int kUnrollSolo = 1;  // k chunks per load block, kNG token groups in one wavefront: this
                                // path is rare in the launches that use it, and a deeper block would
                                // set the register budget (and so the occupancy) of the whole kernel
constexpr int kWaves = 4;       // wavefronts per grouped workgroup: consecutive row tiles of one work unit
constexpr int kNGWide = kUnitTokensGrouped / 16;  // token groups of the widest pass (grouped launch)
static_assert(kNGWide == 8, "the wide staging split gives each thread four of the eight groups");

__device__ inline bf16x8 as_bf16x8(uint4 v) {
    bf16x8 r;
    __builtin_memcpy(&r, &v, 16);
    return r;
}

// Expert weights are read once per layer step and never again from cache:
// stream them with nontemporal loads (measured on MI355X for this access
// pattern, one contiguous block per wavefront: 7.0 TB/s against 6.1 TB/s
// for ordinary loads).
__device__ inline uint4 load_stream(const uint4* p) {
    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
    return uint4{v.x, v.y, v.z, v.w};
}

__device__ inline f32x4 mfma_bf16(uint4 a, uint4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a), as_bf16x8(b), c, 0, 0, 0);
}

__device__ inline float silu_mul(float g, float u) { return g / (1.0f + __expf(-g)) * u; }

__device__ inline uint32_t pack_bf16x2(float lo, float hi) {
    // round to nearest even
    uint32_t a = __float_as_uint(lo), b = __float_as_uint(hi);
    a += 0x7FFFu + ((a >> 16) & 1u);
    b += 0x7FFFu + ((b >> 16) & 1u);
    return (a >> 16) | (b & 0xFFFF0000u);
}

// Gated output of (stream s, slot k) at d-rows j .. j + 3 (c0) and
// j + 16 .. j + 19 (c1), rounded to bf16 like the SwiGLU intermediate: the
// combine adds them in fp32.
__device__ inline void store_gated(const Layout& lo, int s, int k, int j, float gk, const f32x4& c0, const f32x4& c1) {
    uint16_t* dst = reinterpret_cast<uint16_t*>(lo.yp) + ((int64_t)s * lo.K + k) * lo.d + j;
    *reinterpret_cast<uint2*>(dst) = make_uint2(pack_bf16x2(gk * c0[0], gk * c0[1]), pack_bf16x2(gk * c0[2], gk * c0[3]));
    *reinterpret_cast<uint2*>(dst + 16) =
        make_uint2(pack_bf16x2(gk * c1[0], gk * c1[1]), pack_bf16x2(gk * c1[2], gk * c1[3]));
}

// The FFN grids hold wgn workgroups per work unit; consecutive workgroups go
// to the eight XCDs in turn.  With xcd_units, workgroup b takes unit
// u = 8 (q / wgn) + b % 8 and part q % wgn of it, q = b / 8, so that all the
// workgroups of a unit have the same b % 8: a unit runs on one XCD and its
// tokens' activations are fetched into one L2 instead of eight.  Units come
// heaviest first, and each XCD takes every eighth one.  That grid is rounded
// up to whole groups of eight units; u may exceed the last unit.  Without
// it, workgroup b takes unit b / wgn, part b % wgn, and every unit is spread
// over all XCDs: with few tokens per expert there is little to share, and
// whole units per XCD were measured to stream the weights more slowly (up to
// 15% at one token per expert).
__device__ inline void unit_of_block(int b, int wgn, bool xcd, int& u, int& j) {
    if (xcd) {
        const int q = b >> 3, g = q / wgn;
        u = g * 8 + (b & 7);
        j = q - g * wgn;
    } else {
        u = b / wgn;
        j = b - u * wgn;
    }
}

inline int unit_groups(const Layout& lo) { return lo.xcd_units ? (lo.max_units + 7) / 8 * 8 : lo.max_units; }

__device__ inline const uint16_t* slot_base(const Layout& lo, int l, int slot) {
    return reinterpret_cast<const uint16_t*>(lo.arena) + ((int64_t)l * lo.n_slots + slot) * lo.expert_elems;
}

// U consecutive 64-wide k chunks of one 16-row (gate/up) or 2 x 16-row (down)
// weight tile against NG groups of 16 token columns.  All weight and
// activation loads of the block are issued before the first matrix-core
// instruction, so a wavefront waits once per block.  Token columns past the
// bucket (also whole groups past it in the last pass) repeat the bucket's last
// token and their output columns are discarded: column j of the product
// depends on column j of B only.
template <int NG, int U>
__device__ inline void mfma_block(const uint4* __restrict__ tile, int c, const uint16_t* const* xb, f32x4* acc0,
                                  f32x4* acc1) {
    uint4 A[U][4], X[NG][U][2];
#pragma unroll
    for (int i = 0; i < U; ++i) {
        const uint4* ch = tile + (int64_t)(c + i) * 256;
        A[i][0] = load_stream(ch);
        A[i][1] = load_stream(ch + 64);
        A[i][2] = load_stream(ch + 128);
        A[i][3] = load_stream(ch + 192);
    }
#pragma unroll
    for (int q = 0; q < NG; ++q) {
#pragma unroll
        for (int i = 0; i < U; ++i) {
            const int kc = (c + i) * 64;
            X[q][i][0] = *reinterpret_cast<const uint4*>(xb[q] + kc);
            X[q][i][1] = *reinterpret_cast<const uint4*>(xb[q] + kc + 32);
        }
    }
    __builtin_amdgcn_sched_barrier(0);  // keep every load of the block ahead of the matrix-core work
#pragma unroll
    for (int q = 0; q < NG; ++q) {
#pragma unroll
        for (int i = 0; i < U; ++i) {
            acc0[q] = mfma_bf16(A[i][0], X[q][i][0], acc0[q]);
            acc0[q] = mfma_bf16(A[i][1], X[q][i][1], acc0[q]);
            acc1[q] = mfma_bf16(A[i][2], X[q][i][0], acc1[q]);
            acc1[q] = mfma_bf16(A[i][3], X[q][i][1], acc1[q]);
        }
    }
}

// The k loop of one pass: blocks of U chunks, then single chunks.
template <int NG, int U>
__device__ inline void mfma_pass(const uint4* __restrict__ tile, int nchunk, const uint16_t* const* xb, f32x4* acc0,
                                 f32x4* acc1) {
#pragma unroll
    for (int q = 0; q < NG; ++q) {
        acc0[q] = f32x4{0.f, 0.f, 0.f, 0.f};
        acc1[q] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    int c = 0;
    for (; c + U <= nchunk; c += U) mfma_block<NG, U>(tile, c, xb, acc0, acc1);
    for (; c < nchunk; ++c) mfma_block<NG, 1>(tile, c, xb, acc0, acc1);
}

// Grouped launch, units of more than 16 tokens: the kWaves wavefronts of a
// workgroup (row tiles of the same unit) load the activations of each block
// of U k-chunks from global memory once, into LDS, and read their B
// fragments from there.
// Slot (group q, chunk i, half hh) of a buffer holds, for lane (r, g), token
// column r's 8 values at k = 64 (c + i) + 32 hh + 8 g.  Two buffers: one
// barrier per block.
template <int U>
struct HeavyLds {
    uint4 x[2][kNG * U * 2][64];
};
static_assert(kWaves == 4, "the staging split below assumes 4 wavefronts");

// Staging loads of thread tid (U = 2): group q, chunk tid / 128, half
// (tid / 64) % 2, lane tid % 64 for every q, whose token row and k offset are
// the thread's own xb[q] (a chunk past the end is clamped; it is never used).
struct Staged {
    uint4 v[kNG];
};

template <int U>
__device__ inline Staged stage_load(const uint16_t* const* xb, int c, int nchunk, int tid) {
    static_assert(U == 2, "the staging split assumes two chunks per block");
    const int i = tid >> 7, hh = (tid >> 6) & 1;
    const int off = min(c + i, nchunk - 1) * 64 + 32 * hh;
    Staged st;
#pragma unroll
    for (int q = 0; q < kNG; ++q) st.v[q] = *reinterpret_cast<const uint4*>(xb[q] + off);
    return st;
}

// LDS stores of the ng groups in use (wavefront-uniform).
template <int U>
__device__ inline void stage_store(uint4 (*xs)[64], int tid, int ng, const Staged& st) {
    const int i = tid >> 7, hh = (tid >> 6) & 1;
#pragma unroll
    for (int q = 0; q < kNG; ++q)
        if (q < ng) xs[(q * U + i) * 2 + hh][tid & 63] = st.v[q];
}

// One pass of ng (up to kNG) token groups over a 16-row (gate/up) or
// 2 x 16-row (down) weight tile with the activations shared through LDS.
// Every wavefront of the workgroup runs the loop (and its barriers); only
// `active` wavefronts run the matrix-core work.  Every global load is
// unconditional, so that the waits before the LDS stores cover the staging
// loads only: the weight loads of an inactive wavefront re-read its tile's
// first chunk (cached), and staging loads of unused groups repeat the last
// token.
template <int U>
__device__ inline void mfma_pass_shared(const uint4* __restrict__ tile, int nchunk, const uint16_t* const* xb, int ng,
                                        bool active, HeavyLds<U>& sm, int tid, f32x4* acc0, f32x4* acc1) {
    const int lane = tid & 63;
    ng = __builtin_amdgcn_readfirstlane(ng);
#pragma unroll
    for (int q = 0; q < kNG; ++q) {
        acc0[q] = f32x4{0.f, 0.f, 0.f, 0.f};
        acc1[q] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    // The activations of block c + U are loaded while block c computes;
    // their LDS stores then wait only for them, not for the weight loads
    // issued after them.
    Staged st = stage_load<U>(xb, 0, nchunk, tid);
    int b = 0;
    for (int c = 0; c < nchunk; c += U, b ^= 1) {
        uint4 A[U][4];
#pragma unroll
        for (int i = 0; i < U; ++i) {
            const uint4* ch = tile + (int64_t)(active ? min(c + i, nchunk - 1) : 0) * 256;
            A[i][0] = load_stream(ch);
            A[i][1] = load_stream(ch + 64);
            A[i][2] = load_stream(ch + 128);
            A[i][3] = load_stream(ch + 192);
        }
        stage_store<U>(sm.x[b], tid, ng, st);
        __syncthreads();
        st = stage_load<U>(xb, c + U, nchunk, tid);
        if (!active) continue;
#pragma unroll
        for (int q = 0; q < kNG; ++q) {
            if (q >= ng) break;
            uint4 X[U][2];
#pragma unroll
            for (int i = 0; i < U; ++i) {
                X[i][0] = sm.x[b][(q * U + i) * 2][lane];
                X[i][1] = sm.x[b][(q * U + i) * 2 + 1][lane];
            }
#pragma unroll
            for (int i = 0; i < U; ++i) {
                if (c + i < nchunk) {
                    acc0[q] = mfma_bf16(A[i][0], X[i][0], acc0[q]);
                    acc0[q] = mfma_bf16(A[i][1], X[i][1], acc0[q]);
                    acc1[q] = mfma_bf16(A[i][2], X[i][0], acc1[q]);
                    acc1[q] = mfma_bf16(A[i][3], X[i][1], acc1[q]);
                }
            }
        }
    }
}

// Grouped launch, units of 65 to kUnitTokensGrouped tokens (a hot expert's
// tokens in one pass, so its weights are streamed once): the activations of
// one k chunk for all eight token groups (16 KB) are staged in LDS once per
// workgroup, two buffers, one barrier per chunk.  Slot (group q, half hh)
// holds, for lane (r, g), token column r's 8 values at k = 64 c + 32 hh + 8 g.
// Its 32 KB share the workgroup's LDS with HeavyLds.
struct WideLds {
    uint4 x[2][kNGWide * 2][64];
};
union GroupedLds {
    HeavyLds<kUnrollWide> narrow;
    WideLds wide;
};

// Staging of thread tid: groups 4 (tid / 128) .. + 3 at half (tid / 64) % 2
// of chunk c (clamped; a chunk past the end is never used), from the token
// rows xs of those four groups.
__device__ __forceinline__ Staged wide_stage_load(const uint16_t* const* xs, int c, int nchunk, int tid) {
    const int off = min(c, nchunk - 1) * 64 + 32 * ((tid >> 6) & 1);
    Staged st;
#pragma unroll
    for (int q = 0; q < 4; ++q) st.v[q] = *reinterpret_cast<const uint4*>(xs[q] + off);
    return st;
}

__device__ __forceinline__ void wide_stage_store(uint4 (*xb)[64], int tid, int ng, const Staged& st) {
    const int q0 = 4 * (tid >> 7), hh = (tid >> 6) & 1;
#pragma unroll
    for (int q = 0; q < 4; ++q)
        if (q0 + q < ng) xb[(q0 + q) * 2 + hh][tid & 63] = st.v[q];
}

// One pass of ng (up to 8) token groups over a 16-row (gate/up) or 2 x 16-row
// (down) weight tile, the activations shared through LDS, one k chunk per
// block: the next chunk's weights are loaded while the current one computes.
// As in the four-group pass, every wavefront runs the loop and its barriers
// and every global load is unconditional; only `active` wavefronts compute.
__device__ __forceinline__ void mfma_pass_wide(const uint4* __restrict__ tile, int nchunk, const uint16_t* const* xs, int ng,
                                      bool active, WideLds& sm, int tid, f32x4* acc0, f32x4* acc1) {
    const int lane = tid & 63;
    ng = __builtin_amdgcn_readfirstlane(ng);
#pragma unroll
    for (int q = 0; q < kNGWide; ++q) {
        acc0[q] = f32x4{0.f, 0.f, 0.f, 0.f};
        acc1[q] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    Staged st = wide_stage_load(xs, 0, nchunk, tid);
    int b = 0;
    for (int c = 0; c < nchunk; ++c, b ^= 1) {
        uint4 A[4];
        const uint4* ch = tile + (int64_t)(active ? c : 0) * 256;
#pragma unroll
        for (int j = 0; j < 4; ++j) A[j] = load_stream(ch + 64 * j);
        wide_stage_store(sm.x[b], tid, ng, st);
        __syncthreads();
        st = wide_stage_load(xs, c + 1, nchunk, tid);
        if (active) {
#pragma unroll
            for (int q = 0; q < kNGWide; ++q) {
                if (q >= ng) break;
                const uint4 X0 = sm.x[b][q * 2][lane], X1 = sm.x[b][q * 2 + 1][lane];
                acc0[q] = mfma_bf16(A[0], X0, acc0[q]);
                acc0[q] = mfma_bf16(A[1], X1, acc0[q]);
                acc1[q] = mfma_bf16(A[2], X0, acc1[q]);
                acc1[q] = mfma_bf16(A[3], X1, acc1[q]);
            }
        }
    }
}

// ---------------------------------------------------------------- bf16
// Token groups of one pass over the weights: one group (up to 16 tokens, the
// common case) with a deep k block, or kNG groups with a shallower one.
template <int NG, int U>
__device__ inline void up_passes(const Layout& lo, int l, int ft, const int32_t* __restrict__ bk, int m,
                                 const uint4* __restrict__ tileA, const uint16_t* __restrict__ h, int lane) {
    const int r = lane & 15, g = lane >> 4;
    const int d = lo.d;
    uint16_t* act = reinterpret_cast<uint16_t*>(lo.act);
    for (int t0 = 0; t0 < m; t0 += 16 * NG) {
        const int ng = min(NG, (m - t0 + 15) / 16);
        int pr[NG];
        const uint16_t* xb[NG];
#pragma unroll
        for (int q = 0; q < NG; ++q) pr[q] = bk[min(t0 + 16 * q + r, m - 1)];
#pragma unroll
        for (int q = 0; q < NG; ++q) xb[q] = h + ((int64_t)(pr[q] >> 8) * lo.L + l) * d + 8 * g;
        f32x4 cg[NG], cu[NG];
        mfma_pass<NG, U>(tileA, d / 64, xb, cg, cu);
        // D[i][j]: row i = 4 g + rr of this 16-row tile, token column j = r
#pragma unroll
        for (int q = 0; q < NG; ++q) {
            if (q >= ng) break;
            const int tok = t0 + 16 * q + r;
            if (tok < m) {
                uint2 o;
                o.x = pack_bf16x2(silu_mul(cg[q][0], cu[q][0]), silu_mul(cg[q][1], cu[q][1]));
                o.y = pack_bf16x2(silu_mul(cg[q][2], cu[q][2]), silu_mul(cg[q][3], cu[q][3]));
                const int pair = pr[q];
                const int64_t row = (int64_t)(pair >> 8) * lo.K + (pair & 255);  // token (s, k)
                *reinterpret_cast<uint2*>(act + row * lo.F + ft * 16 + 4 * g) = o;
            }
        }
    }
}

// A unit of 17 to 16 kNG tokens: one pass with the activations shared by the
// workgroup.
__device__ inline void up_heavy(const Layout& lo, int l, int ft, const int32_t* __restrict__ bk, int m,
                                const uint4* __restrict__ tileA, const uint16_t* __restrict__ h, int tid,
                                HeavyLds<kUnrollWide>& sm) {
    const int lane = tid & 63, r = lane & 15, g = lane >> 4;
    const int d = lo.d;
    uint16_t* act = reinterpret_cast<uint16_t*>(lo.act);
    int pr[kNG];
    const uint16_t* xb[kNG];
#pragma unroll
    for (int q = 0; q < kNG; ++q) pr[q] = bk[min(16 * q + r, m - 1)];
#pragma unroll
    for (int q = 0; q < kNG; ++q) xb[q] = h + ((int64_t)(pr[q] >> 8) * lo.L + l) * d + 8 * g;
    f32x4 cg[kNG], cu[kNG];
    mfma_pass_shared<kUnrollWide>(tileA, d / 64, xb, (m + 15) / 16, true, sm, tid, cg, cu);
#pragma unroll
    for (int q = 0; q < kNG; ++q) {
        const int tok = 16 * q + r;
        if (tok < m) {
            uint2 o;
            o.x = pack_bf16x2(silu_mul(cg[q][0], cu[q][0]), silu_mul(cg[q][1], cu[q][1]));
            o.y = pack_bf16x2(silu_mul(cg[q][2], cu[q][2]), silu_mul(cg[q][3], cu[q][3]));
            const int pair = pr[q];
            const int64_t row = (int64_t)(pair >> 8) * lo.K + (pair & 255);
            *reinterpret_cast<uint2*>(act + row * lo.F + ft * 16 + 4 * g) = o;
        }
    }
}

// A unit of 65 to kUnitTokensGrouped tokens: one pass, eight token groups,
// the activations shared by the workgroup.
__device__ __forceinline__ void up_heavy_wide(const Layout& lo, int l, int ft, const int32_t* __restrict__ bk, int m,
                                     const uint4* __restrict__ tileA, const uint16_t* __restrict__ h, int tid,
                                     WideLds& sm) {
    const int lane = tid & 63, r = lane & 15, g = lane >> 4;
    const int d = lo.d, q0 = 4 * (tid >> 7);
    uint16_t* act = reinterpret_cast<uint16_t*>(lo.act);
    const uint16_t* xs[4];  // token rows of this thread's staging groups
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int p = bk[min(16 * (q0 + q) + r, m - 1)];
        xs[q] = h + ((int64_t)(p >> 8) * lo.L + l) * d + 8 * g;
    }
    f32x4 cg[kNGWide], cu[kNGWide];
    mfma_pass_wide(tileA, d / 64, xs, (m + 15) / 16, true, sm, tid, cg, cu);
#pragma unroll
    for (int q = 0; q < kNGWide; ++q) {
        const int tok = 16 * q + r;
        if (tok < m) {
            uint2 o;
            o.x = pack_bf16x2(silu_mul(cg[q][0], cu[q][0]), silu_mul(cg[q][1], cu[q][1]));
            o.y = pack_bf16x2(silu_mul(cg[q][2], cu[q][2]), silu_mul(cg[q][3], cu[q][3]));
            const int pair = bk[tok];
            const int64_t row = (int64_t)(pair >> 8) * lo.K + (pair & 255);
            *reinterpret_cast<uint2*>(act + row * lo.F + ft * 16 + 4 * g) = o;
        }
    }
}

// Work unit u (the fill kernel lays them out, heaviest first) = tokens
// [ut p, ut (p + 1)) of expert e's bucket, ut = lo.unit_tokens; workgroup
// (u, j) runs that pass for the W 16-row F-tiles W j + wavefront (F is a
// multiple of 64, so every wavefront has a tile).  W = 1: every wavefront
// on its own; W = kWaves: grouped.
template <int W>
__global__ __launch_bounds__(64 * W) __attribute__((amdgpu_waves_per_eu(3))) void ffn_up_bf16(Layout lo, int l, int bbuf, int /*sv: slots come with the units*/,
                                                      const uint16_t* __restrict__ h) {
    const int wgn = lo.F / (16 * W);
    int u, j;
    unit_of_block(blockIdx.x, wgn, lo.xcd_units != 0, u, j);
    if (u >= lo.max_units) return;
    const int lane = threadIdx.x & 63;
    const int ft = j * W + (threadIdx.x >> 6);
    const int4 ui = reinterpret_cast<const int4*>(lo.units)[u];  // expert, pass, slot, tokens in one load
    if (ui.x < 0) return;
    const int e = ui.x & 255, t0 = lo.unit_tokens * (ui.x >> 8), slot = ui.y, m = ui.z;
    if (m <= 0 || slot < 0 || slot >= lo.n_slots) return;
    const int32_t* bk = lo.pairs + ((int64_t)bbuf * lo.N + e) * lo.S + t0;
    // packed slot layout: chunk c of this row tile is 256 units of 16 bytes,
    // gate half 0, gate half 1, up half 0, up half 1, each 64 units
    const uint4* tileA =
        reinterpret_cast<const uint4*>(slot_base(lo, l, slot)) + (int64_t)ft * (lo.d / 64) * 256 + lane;
    if (m <= 16) {  // workgroup-uniform
        up_passes<1, kUnroll>(lo, l, ft, bk, m, tileA, h, lane);
    } else if constexpr (W == 1) {
        up_passes<kNG, kUnrollSolo>(lo, l, ft, bk, m, tileA, h, lane);
    } else {
        __shared__ GroupedLds sm;
        if (m <= 16 * kNG)
            up_heavy(lo, l, ft, bk, m, tileA, h, threadIdx.x, sm.narrow);
        else
            up_heavy_wide(lo, l, ft, bk, m, tileA, h, threadIdx.x, sm.wide);
    }
}

template <int NG, int U>
__device__ inline void down_passes(const Layout& lo, int l, int dt, const int32_t* __restrict__ bk, int m,
                                   const uint4* __restrict__ tileB, int lane) {
    const int r = lane & 15, g = lane >> 4;
    const int F = lo.F;
    const uint16_t* act = reinterpret_cast<const uint16_t*>(lo.act);
    for (int t0 = 0; t0 < m; t0 += 16 * NG) {
        const int ng = min(NG, (m - t0 + 15) / 16);
        int pr[NG];
        const uint16_t* xb[NG];
#pragma unroll
        for (int q = 0; q < NG; ++q) pr[q] = bk[min(t0 + 16 * q + r, m - 1)];
#pragma unroll
        for (int q = 0; q < NG; ++q) xb[q] = act + ((int64_t)(pr[q] >> 8) * lo.K + (pr[q] & 255)) * F + 8 * g;
        f32x4 c0[NG], c1[NG];
        mfma_pass<NG, U>(tileB, F / 64, xb, c0, c1);
#pragma unroll
        for (int q = 0; q < NG; ++q) {
            if (q >= ng) break;
            const int tok = t0 + 16 * q + r;
            if (tok < m) {
                const int s = pr[q] >> 8, k = pr[q] & 255;
                const float gk = lo.gates[((int64_t)l * lo.S + s) * lo.K + k];
                store_gated(lo, s, k, dt * 32 + 4 * g, gk, c0[q], c1[q]);
            }
        }
    }
}

// A unit of 17 to 16 kNG tokens in the grouped launch: one pass with
// the SwiGLU intermediate shared by the workgroup.  Wavefronts past the last
// d-tile (d not a multiple of 32 W) take part in the staging and barriers
// only.
__device__ inline void down_heavy(const Layout& lo, int l, int dt, bool active, const int32_t* __restrict__ bk, int m,
                                  const uint4* __restrict__ tileB, int tid, HeavyLds<kUnrollWide>& sm) {
    const int lane = tid & 63, r = lane & 15, g = lane >> 4;
    const int F = lo.F;
    const uint16_t* act = reinterpret_cast<const uint16_t*>(lo.act);
    int pr[kNG];
    const uint16_t* xb[kNG];
#pragma unroll
    for (int q = 0; q < kNG; ++q) pr[q] = bk[min(16 * q + r, m - 1)];
#pragma unroll
    for (int q = 0; q < kNG; ++q) xb[q] = act + ((int64_t)(pr[q] >> 8) * lo.K + (pr[q] & 255)) * F + 8 * g;
    f32x4 c0[kNG], c1[kNG];
    mfma_pass_shared<kUnrollWide>(tileB, F / 64, xb, (m + 15) / 16, active, sm, tid, c0, c1);
    if (!active) return;
#pragma unroll
    for (int q = 0; q < kNG; ++q) {
        const int tok = 16 * q + r;
        if (tok < m) {
            const int s = pr[q] >> 8, k = pr[q] & 255;
            const float gk = lo.gates[((int64_t)l * lo.S + s) * lo.K + k];
            store_gated(lo, s, k, dt * 32 + 4 * g, gk, c0[q], c1[q]);
        }
    }
}

// A unit of 65 to kUnitTokensGrouped tokens in the grouped launch: one pass,
// eight token groups, the SwiGLU intermediate shared by the workgroup.
__device__ __forceinline__ void down_heavy_wide(const Layout& lo, int l, int dt, bool active, const int32_t* __restrict__ bk,
                                       int m, const uint4* __restrict__ tileB, int tid, WideLds& sm) {
    const int lane = tid & 63, r = lane & 15, g = lane >> 4;
    const int F = lo.F, q0 = 4 * (tid >> 7);
    const uint16_t* act = reinterpret_cast<const uint16_t*>(lo.act);
    const uint16_t* xs[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int p = bk[min(16 * (q0 + q) + r, m - 1)];
        xs[q] = act + ((int64_t)(p >> 8) * lo.K + (p & 255)) * F + 8 * g;
    }
    f32x4 c0[kNGWide], c1[kNGWide];
    mfma_pass_wide(tileB, F / 64, xs, (m + 15) / 16, active, sm, tid, c0, c1);
    if (!active) return;
#pragma unroll
    for (int q = 0; q < kNGWide; ++q) {
        const int tok = 16 * q + r;
        if (tok < m) {
            const int pair = bk[tok];
            const int s = pair >> 8, k = pair & 255;
            const float gk = lo.gates[((int64_t)l * lo.S + s) * lo.K + k];
            store_gated(lo, s, k, dt * 32 + 4 * g, gk, c0[q], c1[q]);
        }
    }
}

// Workgroup (u, j): the W 32-row d-tiles W j + wavefront of unit u.
template <int W>
__global__ __launch_bounds__(64 * W) __attribute__((amdgpu_waves_per_eu(3))) void ffn_down_bf16(Layout lo, int l, int bbuf, int /*sv: slots come with the units*/) {
    const int dtn = lo.d / 32;
    const int wgn = (dtn + W - 1) / W;
    int u, j;
    unit_of_block(blockIdx.x, wgn, lo.xcd_units != 0, u, j);
    if (u >= lo.max_units) return;
    const int lane = threadIdx.x & 63;
    const int dt = j * W + (threadIdx.x >> 6);
    const bool active = dt < dtn;
    const int4 ui = reinterpret_cast<const int4*>(lo.units)[u];  // expert, pass, slot, tokens in one load
    if (ui.x < 0) return;
    const int e = ui.x & 255, t0 = lo.unit_tokens * (ui.x >> 8), slot = ui.y, m = ui.z;
    if (m <= 0 || slot < 0 || slot >= lo.n_slots) return;
    const int32_t* bk = lo.pairs + ((int64_t)bbuf * lo.N + e) * lo.S + t0;
    // packed slot layout: after the gate/up part (F d / 4 units), chunk c of
    // this 32-row tile is 256 units: rows 0-15 half 0, half 1, rows 16-31
    // half 0, half 1, each 64 units
    const uint4* tileB = reinterpret_cast<const uint4*>(slot_base(lo, l, slot)) + (int64_t)lo.F * lo.d / 4 +
                         (int64_t)(active ? dt : 0) * (lo.F / 64) * 256 + lane;
    if (m <= 16) {  // workgroup-uniform; this path has no barriers
        if (active) down_passes<1, kUnroll>(lo, l, dt, bk, m, tileB, lane);
    } else if constexpr (W == 1) {
        down_passes<kNG, kUnrollSolo>(lo, l, dt, bk, m, tileB, lane);
    } else {
        __shared__ GroupedLds sm;
        if (m <= 16 * kNG)
            down_heavy(lo, l, dt, active, bk, m, tileB, threadIdx.x, sm.narrow);
        else
            down_heavy_wide(lo, l, dt, active, bk, m, tileB, threadIdx.x, sm.wide);
    }
}

// ---------------------------------------------------------------- fp32
__global__ __launch_bounds__(64) void ffn_up_f32(Layout lo, int l, int bbuf, int sv, int round,
                                                 const float* __restrict__ h) {
    const int ftn = lo.F / 64;
    const int e = blockIdx.x / ftn, ft = blockIdx.x - e * ftn;
    const int m = lo.bcount[(int64_t)bbuf * lo.N + e];
    if (m == 0 || lo.round_of[e] != round) return;
    const int32_t* bk = lo.pairs + ((int64_t)bbuf * lo.N + e) * lo.S;
    const int slot = lo.slot_of[((int64_t)sv * lo.L + l) * lo.N + e];
    if (slot < 0 || slot >= lo.n_slots) return;
    // transposed in the slot (the fill writes W_gate^T, W_up^T as [d][F]):
    // the 64 lanes, rows f, read 64 consecutive floats per k
    const float* Wg = reinterpret_cast<const float*>(lo.arena) + ((int64_t)l * lo.n_slots + slot) * lo.expert_elems;
    const float* Wu = Wg + (int64_t)lo.F * lo.d;
    const int f = ft * 64 + threadIdx.x;
    float* act = reinterpret_cast<float*>(lo.act);
    for (int tok = 0; tok < m; ++tok) {
        const int pair = bk[tok];
        const int s = pair >> 8;
        const float* x = h + ((int64_t)s * lo.L + l) * lo.d;
        float ag = 0.0f, au = 0.0f;
        for (int i0 = 0; i0 < lo.d; i0 += 32) {  // d is a multiple of 64
            float wg[32], wu[32], xv[32];        // every load of a batch issued before the FMAs
#pragma unroll
            for (int u = 0; u < 32; ++u) {
                wg[u] = Wg[(int64_t)(i0 + u) * lo.F + f];
                wu[u] = Wu[(int64_t)(i0 + u) * lo.F + f];
                xv[u] = x[i0 + u];
            }
#pragma unroll
            for (int u = 0; u < 32; ++u) {
                ag = __builtin_fmaf(wg[u], xv[u], ag);
                au = __builtin_fmaf(wu[u], xv[u], au);
            }
        }
        act[((int64_t)s * lo.K + (pair & 255)) * lo.F + f] = ag / (1.0f + expf(-ag)) * au;
    }
}

__global__ __launch_bounds__(64) void ffn_down_f32(Layout lo, int l, int bbuf, int sv, int round) {
    const int dtn = lo.d / 64;
    const int e = blockIdx.x / dtn, dt = blockIdx.x - e * dtn;
    const int m = lo.bcount[(int64_t)bbuf * lo.N + e];
    if (m == 0 || lo.round_of[e] != round) return;
    const int32_t* bk = lo.pairs + ((int64_t)bbuf * lo.N + e) * lo.S;
    const int slot = lo.slot_of[((int64_t)sv * lo.L + l) * lo.N + e];
    if (slot < 0 || slot >= lo.n_slots) return;
    // W_down^T [F][d] in the slot: lanes (rows j) read consecutive floats
    const float* Wd = reinterpret_cast<const float*>(lo.arena) + ((int64_t)l * lo.n_slots + slot) * lo.expert_elems +
                      2 * (int64_t)lo.F * lo.d;
    const int j = dt * 64 + threadIdx.x;
    const float* act = reinterpret_cast<const float*>(lo.act);
    for (int tok = 0; tok < m; ++tok) {
        const int pair = bk[tok];
        const int s = pair >> 8, k = pair & 255;
        const float* av = act + ((int64_t)s * lo.K + k) * lo.F;
        float acc = 0.0f;
        for (int f0 = 0; f0 < lo.F; f0 += 32) {  // F is a multiple of 64
            float wd[32], a32[32];
#pragma unroll
            for (int u = 0; u < 32; ++u) {
                wd[u] = Wd[(int64_t)(f0 + u) * lo.d + j];
                a32[u] = av[f0 + u];
            }
#pragma unroll
            for (int u = 0; u < 32; ++u) acc = __builtin_fmaf(wd[u], a32[u], acc);
        }
        const float gk = lo.gates[((int64_t)l * lo.S + s) * lo.K + k];
        reinterpret_cast<float*>(lo.yp)[((int64_t)s * lo.K + k) * lo.d + j] = gk * acc;
    }
}

}  // namespace

hipError_t launch_ffn_up(const Layout& lo, int l, int bbuf, int sv, int round, const void* h, hipStream_t st,
                         const Timing& tm) {
    if (lo.dtype == 1) {
        const uint16_t* hb = static_cast<const uint16_t*>(h);
        if (lo.ffn_waves == kWaves)
            launch_kernel(ffn_up_bf16<kWaves>, dim3(unit_groups(lo) * (lo.F / (16 * kWaves))), dim3(64 * kWaves), st, tm,
                          lo, l, bbuf, sv, hb);
        else
            launch_kernel(ffn_up_bf16<1>, dim3(unit_groups(lo) * (lo.F / 16)), dim3(64), st, tm, lo, l, bbuf, sv, hb);
    } else {
        launch_kernel(ffn_up_f32, dim3(lo.N * (lo.F / 64)), dim3(64), st, tm, lo, l, bbuf, sv, round,
                      static_cast<const float*>(h));
    }
    return hipGetLastError();
}

hipError_t launch_ffn_down(const Layout& lo, int l, int bbuf, int sv, int round, hipStream_t st, const Timing& tm) {
    if (lo.dtype == 1) {
        const int dtn = lo.d / 32;
        if (lo.ffn_waves == kWaves)
            launch_kernel(ffn_down_bf16<kWaves>, dim3(unit_groups(lo) * ((dtn + kWaves - 1) / kWaves)), dim3(64 * kWaves),
                          st, tm, lo, l, bbuf, sv);
        else
            launch_kernel(ffn_down_bf16<1>, dim3(unit_groups(lo) * dtn), dim3(64), st, tm, lo, l, bbuf, sv);
    } else {
        launch_kernel(ffn_down_f32, dim3(lo.N * (lo.d / 64)), dim3(64), st, tm, lo, l, bbuf, sv, round);
    }
    return hipGetLastError();
}

}  // namespace cmoe
