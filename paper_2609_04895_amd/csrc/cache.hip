// cache.hip - the per-(stream, layer) cache state machine of the decode step.
//
// cache_step_kernel: one wavefront per stream; expert e of the layer lives in
// lane e % 64, register e / 64.  For the accessed layer l it
//   - finishes the router logits (adds the split-K partials in ascending
//     order, adds the native bias, rounds once to fp32),
//   - computes p^R, p^T (and p^S in full mode) with the fixed fp32 softmax
//     described below (Section 2, Section 3.2, Section 3.3),
//   - selects S = TopK by native logit (ties: lower index) and the gate
//     weights p^R_S / sum p^R_S,
//   - counts hits and demand misses against the resident set (Section 2),
//   - applies the post-access retention update with s^T = p^R + p^T
//     (Algorithm 1: each demand-loaded expert in ascending order fills free
//     room or replaces the lowest-s^T resident that is not selected now;
//     ties evict the lower index),
//   - stores s^T as the next token's a^T (Section 3.3) and p^S as the
//     prediction for the causal successor.
// In full mode it then refines the successor layer's cache before that
// layer is accessed (Algorithm 2): candidates Top_R(s^ST), s^ST = a^T + p^S
// of the causal predecessor, examined in descending order; a non-resident
// candidate fills free room, else replaces the lowest-s^ST resident when its
// score is strictly higher.  The first layer of a token is refined by a
// refine-only launch at the start of the token, from the previous token's
// last-layer p^S (the wrap-around of the causal predecessor).
//
// finish_kernel (one workgroup): for a layer whose caches changed, makes the
// HBM slots hold the union of the streams' caches (experts that left free
// their slots; each new expert, ascending, takes the lowest free slot and is
// queued for a copy from the cold pool), and groups the layer's (stream, k)
// selections by expert for the FFN.
//
// Fixed fp32 softmax: m = max z; u_e = exp(z_e - m) with the exponential
// below; the sum is a strided halving over the next power of two P >= N
// (v[i] += v[i + w] for w = P/2 .. 1, missing entries +0), which maps onto
// in-lane adds for w >= 64 and shuffle-down adds for w < 64; p_e = u_e / sum
// (IEEE division).  exp(x), x <= 0: +0 below -80; else k = rint(x / ln 2),
// r = x - k ln2_hi - k ln2_lo (Cody & Waite; ln2_hi is fl32(ln 2) with the low
// 8 fraction bits cleared, ln2_lo = fl32(ln 2 - ln2_hi)), a degree-7 Taylor
// polynomial in Horner form with coefficients fl32(1/n!), scaled by 2^k.
// Build with -ffp-contract=off: every operation here is rounded separately.
#include <math.h>

#include "cmoe_internal.h"

namespace cmoe {

namespace {

constexpr float kLn2Hi = 0x1.62e4p-1f;       // 0x3f317200
constexpr float kLn2Lo = 0x1.7f7d1cp-20f;    // 0x35bfbe8e
constexpr float kInvLn2 = 0x1.715476p+0f;    // fl32(1 / ln 2)
constexpr float kC0 = 1.0f, kC1 = 1.0f, kC2 = 0.5f;
constexpr float kC3 = 0x1.555556p-3f;        // fl32(1/6)
constexpr float kC4 = 0x1.555556p-5f;        // fl32(1/24)
constexpr float kC5 = 0x1.111112p-7f;        // fl32(1/120)
constexpr float kC6 = 0x1.6c16c2p-10f;       // fl32(1/720)
constexpr float kC7 = 0x1.a01a02p-13f;       // fl32(1/5040)

__device__ inline float canon_exp(float x) {
    if (x < -80.0f) return 0.0f;
    const float k = __builtin_rintf(x * kInvLn2);
    float r = __builtin_fmaf(-k, kLn2Hi, x);
    r = __builtin_fmaf(-k, kLn2Lo, r);
    float p = kC7;
    p = __builtin_fmaf(p, r, kC6);
    p = __builtin_fmaf(p, r, kC5);
    p = __builtin_fmaf(p, r, kC4);
    p = __builtin_fmaf(p, r, kC3);
    p = __builtin_fmaf(p, r, kC2);
    p = __builtin_fmaf(p, r, kC1);
    p = __builtin_fmaf(p, r, kC0);
    return __builtin_ldexpf(p, (int)k);
}

// Order-preserving map of fp32 onto uint32 (larger float -> larger key);
// -0 and +0 map to the same key.
__device__ inline uint32_t ord32(float x) {
    uint32_t u = __float_as_uint(x);
    if ((u & 0x7FFFFFFFu) == 0) u = 0;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ inline unsigned long long wave_max_u64(unsigned long long v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const unsigned long long w = __shfl_xor(v, o);
        v = w > v ? w : v;
    }
    return v;
}

__device__ inline unsigned long long wave_min_u64(unsigned long long v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const unsigned long long w = __shfl_xor(v, o);
        v = w < v ? w : v;
    }
    return v;
}

__device__ inline float wave_max_f32(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
    return v;
}

template <int NPL>
__device__ inline void softmax_fixed(const float (&z)[NPL], int N, int lane, float (&p)[NPL]) {
    float m = -INFINITY;
#pragma unroll
    for (int j = 0; j < NPL; ++j)
        if (j * 64 + lane < N) m = fmaxf(m, z[j]);
    m = wave_max_f32(m);
    float v[NPL];
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
        const bool in = j * 64 + lane < N;
        p[j] = in ? canon_exp(z[j] - m) : 0.0f;
        v[j] = p[j];
    }
    int P = 1;
    while (P < N) P <<= 1;
    // in-lane halving steps (w >= 64)
#pragma unroll
    for (int jw = NPL / 2; jw >= 1; jw >>= 1) {
        if (jw * 64 * 2 <= P) {
#pragma unroll
            for (int j = 0; j < jw; ++j) v[j] = v[j] + v[j + jw];
        }
    }
    // cross-lane halving steps (w < 64)
    float x = v[0];
    for (int w = (P / 2 < 32 ? P / 2 : 32); w >= 1; w >>= 1) {
        const float o = __shfl_down(x, w);
        x = x + o;
    }
    const float sum = __shfl(x, 0);
#pragma unroll
    for (int j = 0; j < NPL; ++j) p[j] = p[j] / sum;
}

template <int NPL>
__device__ inline bool bit_of(const unsigned long long (&w)[NPL], int e) {
    bool b = false;
#pragma unroll
    for (int j = 0; j < NPL; ++j)
        if (j == (e >> 6)) b = (w[j] >> (e & 63)) & 1ull;
    return b;
}

// Lowest-scoring member (bit set in member words) with the lowest index on
// ties; returns (ord(score) << 32) | e, or ~0 if there is no member.
template <int NPL>
__device__ inline unsigned long long argmin_member(const float (&sc)[NPL], const unsigned long long (&member)[NPL],
                                                   int N, int lane) {
    unsigned long long best = ~0ull;
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
        const int e = j * 64 + lane;
        if (e < N && ((member[j] >> lane) & 1ull)) {
            const unsigned long long k = ((unsigned long long)ord32(sc[j]) << 32) | (unsigned)e;
            best = k < best ? k : best;
        }
    }
    return wave_min_u64(best);
}

template <int NPL>
__device__ inline void set_bit(unsigned long long (&w)[NPL], int e) {
#pragma unroll
    for (int j = 0; j < NPL; ++j)
        if (j == (e >> 6)) w[j] |= 1ull << (e & 63);
}

template <int NPL>
__device__ inline void clear_bit(unsigned long long (&w)[NPL], int e) {
#pragma unroll
    for (int j = 0; j < NPL; ++j)
        if (j == (e >> 6)) w[j] &= ~(1ull << (e & 63));
}

// Pre-access refinement of one (stream, layer) cache (Algorithm 2).
template <int NPL>
__device__ void refine_one(const Layout& lo, int s, int rl, int R, bool counted, const float (&pred)[NPL],
                           const float (&aTv)[NPL], const unsigned long long (&cw_in)[NPL], int lane) {
    const int N = lo.N;
    float sST[NPL];
    unsigned long long cand[NPL];
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
        const int e = j * 64 + lane;
        if (e < N) {
            sST[j] = aTv[j] + pred[j];
            cand[j] = ((unsigned long long)ord32(sST[j]) << 32) | (0xFFFFFFFFu - (unsigned)e);
        } else {
            sST[j] = 0.0f;
            cand[j] = 0ull;
        }
    }
    unsigned long long* cptr = lo.cache + ((int64_t)s * lo.L + rl) * lo.NW;
    unsigned long long cw[NPL];
    int count = 0;
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
        cw[j] = cw_in[j];
        count += __popcll(cw[j]);
    }
    int nP = 0;
    const int Rn = R < N ? R : N;
    for (int i = 0; i < Rn; ++i) {
        unsigned long long best = 0ull;
#pragma unroll
        for (int j = 0; j < NPL; ++j) best = cand[j] > best ? cand[j] : best;
        best = wave_max_u64(best);
        const int e = (int)(0xFFFFFFFFu - (unsigned)(best & 0xFFFFFFFFull));
        const uint32_t ord_e = (uint32_t)(best >> 32);
#pragma unroll
        for (int j = 0; j < NPL; ++j)
            if (cand[j] == best) cand[j] = 0ull;  // unique key: only the owner matches
        if (bit_of(cw, e)) continue;              // already resident
        if (count < lo.C) {
            set_bit(cw, e);
            ++count;
            ++nP;
        } else {
            const unsigned long long mn = argmin_member(sST, cw, N, lane);
            const int v = (int)(mn & 0xFFFFFFFFull);
            const uint32_t ord_v = (uint32_t)(mn >> 32);
            if (ord_e > ord_v) {  // strictly higher priority
                clear_bit(cw, v);
                set_bit(cw, e);
                ++nP;
            }
        }
    }
    if (lane == 0) {
        for (int j = 0; j < lo.NW; ++j) cptr[j] = cw[j];
        lo.events[((int64_t)rl * lo.S + s) * 4 + 2] = nP;
        if (counted) lo.ctr[((int64_t)s * lo.L + rl) * kNctr + kCtrP] += nP;
    }
}

template <int NPL>
__device__ void stream_step(const Layout& lo, const StepArgs& a, int s, int lane) {
    const int N = lo.N, L = lo.L, K = lo.K;
    const bool full = lo.mode == 1;
    const bool counted = (a.flags & kFlagCount) != 0;
    float pred[NPL];

    // Loads that do not depend on this token's scores are issued first so
    // that their latencies overlap: the refined layer's a^T and cache words,
    // the accessed layer's cache words.
    float aTv[NPL];
    unsigned long long cw_r[NPL], cw_a[NPL];
    const bool refine = (a.flags & kFlagRefine) != 0;
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
        const int e = j * 64 + lane;
        aTv[j] = (refine && e < N) ? lo.aT[((int64_t)s * L + a.rl) * N + e] : 0.0f;
        cw_r[j] = (refine && j < lo.NW) ? lo.cache[((int64_t)s * L + a.rl) * lo.NW + j] : 0ull;
        cw_a[j] = ((a.flags & kFlagAccess) && j < lo.NW) ? lo.cache[((int64_t)s * L + a.l) * lo.NW + j] : 0ull;
    }

    if (a.flags & kFlagAccess) {
        const int l = a.l;
        const int64_t sl = (int64_t)s * L + l;
        // logits
        float z[3][NPL];
#pragma unroll
        for (int r = 0; r < 3; ++r) {
#pragma unroll
            for (int j = 0; j < NPL; ++j) {
                z[r][j] = 0.0f;
                if (r >= lo.n_r) continue;
                const int e = j * 64 + lane;
                float v = 0.0f;
                if (e < N) {
                    if (a.flags & kFlagInject) {
                        const float* src = r == 0 ? a.zR : (r == 1 ? a.zT : a.zS);
                        v = src[sl * N + e];
                    } else {
                        v = lo.logits[(((int64_t)l * lo.S + s) * lo.n_r + r) * N + e];  // router output
                    }
                    if (a.flags & kFlagInject) lo.logits[(((int64_t)l * lo.S + s) * lo.n_r + r) * N + e] = v;
                }
                z[r][j] = v;
            }
        }
        float pR[NPL], pT[NPL];
        softmax_fixed<NPL>(z[0], N, lane, pR);
        softmax_fixed<NPL>(z[1], N, lane, pT);
        if (full) softmax_fixed<NPL>(z[2], N, lane, pred);

        // Top-K by native logit, lower index first on ties
        unsigned long long key[NPL];
#pragma unroll
        for (int j = 0; j < NPL; ++j) {
            const int e = j * 64 + lane;
            key[j] = e < N ? (((unsigned long long)ord32(z[0][j]) << 32) | (0xFFFFFFFFu - (unsigned)e)) : 0ull;
        }
        unsigned long long sw[NPL];
#pragma unroll
        for (int j = 0; j < NPL; ++j) sw[j] = 0ull;
        float gsum = 0.0f, my_p = 0.0f;
        int my_sel = 0;
        for (int k = 0; k < K; ++k) {
            unsigned long long best = 0ull;
#pragma unroll
            for (int j = 0; j < NPL; ++j) best = key[j] > best ? key[j] : best;
            best = wave_max_u64(best);
            const int e = (int)(0xFFFFFFFFu - (unsigned)(best & 0xFFFFFFFFull));
            float pv = 0.0f;
#pragma unroll
            for (int j = 0; j < NPL; ++j) {
                if (key[j] == best) {
                    key[j] = 0ull;
                    pv = pR[j];
                }
            }
            pv = __shfl(pv, e & 63);
            gsum = gsum + pv;
            set_bit(sw, e);
            if (lane == k) {
                my_p = pv;
                my_sel = e;
            }
        }
        if (lane < K) {
            const int64_t o = ((int64_t)l * lo.S + s) * K + lane;
            lo.sel[o] = my_sel;
            lo.gates[o] = my_p / gsum;
        }
        float sT[NPL];
#pragma unroll
        for (int j = 0; j < NPL; ++j) sT[j] = pR[j] + pT[j];

        // access
        unsigned long long* cptr = lo.cache + sl * lo.NW;
        unsigned long long cw[NPL];
        int count = 0, hits = 0;
#pragma unroll
        for (int j = 0; j < NPL; ++j) {
            cw[j] = cw_a[j];
            count += __popcll(cw[j]);
            hits += __popcll(cw[j] & sw[j]);
        }
        const int nD = K - hits;
        // Algorithm 1 with the demand set D = S \ C taken before any insertion
#pragma unroll
        for (int j = 0; j < NPL; ++j) {
            unsigned long long dw = sw[j] & ~cw[j];
            while (dw) {
                const int b = __builtin_ctzll(dw);
                dw &= dw - 1;
                const int e = j * 64 + b;
                if (count < lo.C) {
                    cw[j] |= 1ull << b;
                    ++count;
                } else {
                    unsigned long long vict[NPL];
#pragma unroll
                    for (int jj = 0; jj < NPL; ++jj) vict[jj] = cw[jj] & ~sw[jj];
                    const unsigned long long mn = argmin_member(sT, vict, N, lane);
                    clear_bit(cw, (int)(mn & 0xFFFFFFFFull));
                    cw[j] |= 1ull << b;
                }
            }
        }
        if (lane == 0) {
            for (int j = 0; j < lo.NW; ++j) {
                cptr[j] = cw[j];
                lo.sel_mask[(int64_t)s * lo.NW + j] = sw[j];
            }
            int32_t* ev = lo.events + ((int64_t)l * lo.S + s) * 4;
            ev[0] = hits;
            ev[1] = nD;
            if (!(a.flags & kFlagRefinedHere)) ev[2] = 0;
            ev[3] = 0;
            if (counted) {
                int64_t* c = lo.ctr + sl * kNctr;
                c[kCtrA] += K;
                c[kCtrHits] += hits;
                c[kCtrD] += nD;
                c[kCtrT] += 1;
            }
        }
        if (full) {
#pragma unroll
            for (int j = 0; j < NPL; ++j) {
                const int e = j * 64 + lane;
                if (e < N) {
                    lo.aT[sl * N + e] = sT[j];
                    lo.pS[(int64_t)s * N + e] = pred[j];
                }
            }
        }
    } else {
        // refine-only launch: the predecessor's prediction is the stored one
#pragma unroll
        for (int j = 0; j < NPL; ++j) {
            const int e = j * 64 + lane;
            pred[j] = e < N ? lo.pS[(int64_t)s * N + e] : 0.0f;
        }
    }
    if (refine) refine_one<NPL>(lo, s, a.rl, a.R, counted, pred, aTv, cw_r, lane);
}

template <int NPL>
__global__ __launch_bounds__(256) void cache_step_kernel(Layout lo, StepArgs a) {
    const int lane = threadIdx.x & 63;
    const int s = blockIdx.x * kStreamsPerBlock + (threadIdx.x >> 6);
    if (s < lo.S) stream_step<NPL>(lo, a, s, lane);  // wave-uniform branch
}

// ---------------------------------------------------------------- finish
// Exclusive prefix sum over the 256 threads of the block; *total gets the sum.
__device__ int block_scan(int v, int* total, int* lds4) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    int x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(x, o);
        if (lane >= o) x += y;
    }
    if (lane == 63) lds4[w] = x;
    __syncthreads();
    int off = 0, tot = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        if (i < w) off += lds4[i];
        tot += lds4[i];
    }
    __syncthreads();
    *total = tot;
    return off + x - v;
}

// Staged inputs of finish_kernel in (dynamic) LDS; sizes from finish_lds_bytes.
struct FinishLds {
    unsigned long long* cw_a;  // [S][NW] caches of the accessed layer after retention
    unsigned long long* cw_r;  // [S][NW] caches of the refined layer
    unsigned long long* selm;  // [S][NW] selection masks of the accessed layer
    int* ssel;                 // [S][K]  selection lists of the accessed layer
    int* so_a;                 // [N]     slot of each expert, accessed layer
    int* se_a;                 // [n_slots]
    int* so_r;                 // [N]     refined layer
    int* se_r;                 // [n_slots]
};

__device__ FinishLds carve(const Layout& lo, unsigned char* base) {
    FinishLds f;
    const size_t w = (size_t)lo.S * lo.NW * 8;
    f.cw_a = reinterpret_cast<unsigned long long*>(base);
    f.cw_r = reinterpret_cast<unsigned long long*>(base + w);
    f.selm = reinterpret_cast<unsigned long long*>(base + 2 * w);
    f.ssel = reinterpret_cast<int*>(base + 3 * w);
    f.so_a = f.ssel + (size_t)lo.S * lo.K;
    f.se_a = f.so_a + lo.N;
    f.so_r = f.se_a + lo.n_slots;
    f.se_r = f.so_r + lo.N;
    return f;
}

// Residency event of one layer from the staged caches and slot maps: the
// layer's slots must hold the union U of the streams' caches.  Experts that
// left U free their slot; each new expert (ascending) takes the lowest free
// slot and is queued for a copy from the cold pool.
__device__ void residency(const Layout& lo, int layer, int kind, bool counted, const unsigned long long* cw,
                          int* so, int* se) {
    __shared__ unsigned long long U[4];
    __shared__ int free_list[kMaxN];
    __shared__ int lds4[4];
    const int tid = threadIdx.x;
    if (tid < 4) U[tid] = 0ull;
    __syncthreads();
    for (int i = tid; i < lo.S * lo.NW; i += blockDim.x) {
        const unsigned long long w = cw[i];
        if (w) atomicOr(&U[i % lo.NW], w);
    }
    __syncthreads();
    const int e = tid;
    const bool inU = e < lo.N && ((U[e >> 6] >> (e & 63)) & 1ull);
    int cur = e < lo.N ? so[e] : -1;
    if (e < lo.N && cur >= 0 && !inU) {  // left every cache: free its slot
        se[cur] = -1;
        so[e] = -1;
        cur = -1;
    }
    __syncthreads();
    const bool enter = e < lo.N && inU && cur < 0;
    const bool is_free = tid < lo.n_slots && se[tid] == -1;
    int nfree, nenter;
    const int rf = block_scan(is_free ? 1 : 0, &nfree, lds4);
    if (is_free) free_list[rf] = tid;
    const int re = block_scan(enter ? 1 : 0, &nenter, lds4);
    __syncthreads();
    if (enter) {  // rank re among new experts takes the rank-re free slot
        const int q = free_list[re];
        so[e] = q;
        se[q] = e;
        int32_t* fl = lo.fill_list + (((int64_t)layer * 2 + kind) * lo.N + re) * 2;
        fl[0] = e;
        fl[1] = q;
    }
    __syncthreads();
    if (e < lo.N) lo.slot_of[(int64_t)layer * lo.N + e] = so[e];
    if (tid < lo.n_slots) lo.slot_exp[(int64_t)layer * lo.n_slots + tid] = se[tid];
    if (tid == 0) {
        lo.fill_count[layer * 2 + kind] = nenter;
        lo.step_fills[layer * 2 + kind] = nenter;
        if (counted) lo.phys[layer * 2 + kind] += nenter;
    }
}

// Groups the layer's (stream, k) selections by expert: per expert the token
// count, the first bucket position (exclusive scan over experts), the active
// expert list, and the bucket entries (stream << 8) | k in ascending stream
// order.  Thread e handles expert e, reading the staged masks and lists.
__device__ void buckets(const Layout& lo, int l, bool counted, const unsigned long long* selm, const int* ssel) {
    __shared__ int lds4[4];
    const int e = threadIdx.x;
    const int NW = lo.NW, K = lo.K;
    int cnt = 0;
    if (e < lo.N)
        for (int s = 0; s < lo.S; ++s) cnt += (int)((selm[s * NW + (e >> 6)] >> (e & 63)) & 1ull);
    int total, nact;
    const int off = block_scan(cnt, &total, lds4);
    const int ra = block_scan(cnt > 0 ? 1 : 0, &nact, lds4);
    if (e < lo.N) {
        lo.bcount[e] = cnt;
        lo.boffset[e] = off;
        if (cnt > 0) lo.active[ra] = e;
    }
    if (threadIdx.x == 0) {
        *lo.n_active = nact;
        if (counted) lo.active_sum[l] += nact;
    }
    if (e < lo.N && cnt > 0) {
        int pos = off;
        for (int s = 0; s < lo.S; ++s) {
            if ((selm[s * NW + (e >> 6)] >> (e & 63)) & 1ull) {
                int k = 0;  // rank of e in the stream's selection (it is one of the K)
                for (int kk = 0; kk < K; ++kk)
                    if (ssel[s * K + kk] == e) k = kk;
                lo.pairs[pos++] = (s << 8) | k;
            }
        }
    }
}

__global__ __launch_bounds__(256) void finish_kernel(Layout lo, StepArgs a) {
    extern __shared__ unsigned char finish_lds[];
    const FinishLds f = carve(lo, finish_lds);
    const bool counted = (a.flags & kFlagCount) != 0;
    const bool acc = (a.flags & kFlagAccess) != 0, ref = (a.flags & kFlagRefine) != 0;
    const int tid = threadIdx.x;
    // one parallel staging phase: every input of the kernel into LDS
    const int nw = lo.S * lo.NW;
    for (int i = tid; i < nw; i += blockDim.x) {
        const int s = i / lo.NW, j = i - s * lo.NW;
        if (acc) {
            f.cw_a[i] = lo.cache[((int64_t)s * lo.L + a.l) * lo.NW + j];
            f.selm[i] = lo.sel_mask[i];
        }
        if (ref) f.cw_r[i] = lo.cache[((int64_t)s * lo.L + a.rl) * lo.NW + j];
    }
    if (acc)
        for (int i = tid; i < lo.S * lo.K; i += blockDim.x) f.ssel[i] = lo.sel[(int64_t)a.l * lo.S * lo.K + i];
    if (tid < lo.N) {
        if (acc) f.so_a[tid] = lo.slot_of[(int64_t)a.l * lo.N + tid];
        if (ref) f.so_r[tid] = lo.slot_of[(int64_t)a.rl * lo.N + tid];
    }
    if (tid < lo.n_slots) {
        if (acc) f.se_a[tid] = lo.slot_exp[(int64_t)a.l * lo.n_slots + tid];
        if (ref) f.se_r[tid] = lo.slot_exp[(int64_t)a.rl * lo.n_slots + tid];
    }
    __syncthreads();
    if (acc) {
        residency(lo, a.l, 0, counted, f.cw_a, f.so_a, f.se_a);
        __syncthreads();
        buckets(lo, a.l, counted, f.selm, f.ssel);
        if (tid == 0 && !(a.flags & kFlagRefinedHere)) lo.step_fills[a.l * 2 + 1] = 0;
        __syncthreads();
    }
    if (ref) residency(lo, a.rl, 1, counted, f.cw_r, f.so_r, f.se_r);
}

// ---------------------------------------------------------------- init
__global__ void init_kernel(Layout lo) {
    const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t gs = (int64_t)gridDim.x * blockDim.x;
    const int64_t nc = (int64_t)lo.S * lo.L * lo.NW;
    for (int64_t i = gid; i < nc; i += gs) lo.cache[i] = 0ull;
    const int64_t na = (int64_t)lo.S * lo.L * lo.N;
    for (int64_t i = gid; i < na; i += gs) lo.aT[i] = 0.0f;
    for (int64_t i = gid; i < (int64_t)lo.S * lo.N; i += gs) lo.pS[i] = 0.0f;
    for (int64_t i = gid; i < (int64_t)lo.S * lo.L * kNctr; i += gs) lo.ctr[i] = 0;
    for (int64_t i = gid; i < (int64_t)lo.L * 2; i += gs) {
        lo.phys[i] = 0;
        lo.step_fills[i] = 0;
        if (i < lo.L) lo.active_sum[i] = 0;
        lo.fill_count[i] = 0;
    }
    for (int64_t i = gid; i < (int64_t)lo.L * lo.N; i += gs) lo.slot_of[i] = -1;
    for (int64_t i = gid; i < (int64_t)lo.L * lo.n_slots; i += gs) lo.slot_exp[i] = -1;
    for (int64_t i = gid; i < (int64_t)lo.L * lo.S * 4; i += gs) lo.events[i] = 0;
    for (int64_t i = gid; i < lo.n_tiles; i += gs) lo.tile_count[i] = 0u;
}

}  // namespace

hipError_t launch_init(const Layout& lo, hipStream_t st) {
    hipLaunchKernelGGL(init_kernel, dim3(256), dim3(256), 0, st, lo);
    return hipGetLastError();
}

hipError_t launch_cache_step(const Layout& lo, const StepArgs& a, hipStream_t st) {
    const dim3 grid((lo.S + kStreamsPerBlock - 1) / kStreamsPerBlock);
    if (lo.N <= 64)
        hipLaunchKernelGGL(cache_step_kernel<1>, grid, dim3(256), 0, st, lo, a);
    else if (lo.N <= 128)
        hipLaunchKernelGGL(cache_step_kernel<2>, grid, dim3(256), 0, st, lo, a);
    else
        hipLaunchKernelGGL(cache_step_kernel<4>, grid, dim3(256), 0, st, lo, a);
    return hipGetLastError();
}

size_t finish_lds_bytes(const Layout& lo) {
    return (size_t)lo.S * lo.NW * 8 * 3 + (size_t)lo.S * lo.K * 4 + (size_t)(lo.N + lo.n_slots) * 2 * 4;
}

hipError_t launch_finish(const Layout& lo, const StepArgs& a, hipStream_t st) {
    hipLaunchKernelGGL(finish_kernel, dim3(1), dim3(256), finish_lds_bytes(lo), st, lo, a);
    return hipGetLastError();
}

}  // namespace cmoe
