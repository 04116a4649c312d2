// cache.hip - the per-(stream, layer) cache state machine of the decode step.
//
// cache_step_kernel: one wavefront per stream; expert e of the layer lives in
// lane e % 64, register e / 64.  For the accessed layer l it
//   - finishes the router logits (adds the split-K partials in ascending
//     order, adds the native bias, rounds once to fp32),
//   - computes p^R, p^T (router policy) and p^S (modes with a Spatio
//     Router) with the fixed fp32 softmax described below (Section 2,
//     Section 3.2, Section 3.3),
//   - selects S = TopK by native logit (ties: lower index) and the gate
//     weights p^R_S / sum p^R_S,
//   - counts hits and demand misses against the resident set (Section 2),
//   - applies the post-access retention update (Algorithm 1: each
//     demand-loaded expert in ascending order fills free room or replaces
//     the lowest-priority resident that is not selected now; ties evict the
//     lower index), with priority s^T = p^R + p^T or, for the classical
//     cache-update baselines (Section 4.1, Table 1), the LRU time, LFU count
//     or LRFU value, updated first,
//   - stores the next token's a-score (Section 3.3: s^T in the full mode;
//     p^R in the Spatio-only ablation of Section 5 / Appendix B.4) and p^S
//     as the prediction for the causal successor.
// In the modes with a Spatio Router it then refines the successor layer's
// cache before that layer is accessed (Algorithm 2): candidates Top_R(s^ST),
// s^ST = a + p^S of the causal predecessor, examined in descending order; a
// non-resident candidate fills free room, else replaces the lowest-s^ST
// resident when its score is strictly higher (an inserted expert takes the
// LRU time of the refinement).  The first layer of a token is refined by a
// refine-only launch at the start of the token, from the previous token's
// last-layer p^S (the wrap-around of the causal predecessor).
//
// The same kernel groups the layer's (stream, k) selections by expert for the
// FFN (fixed-capacity buckets filled with integer atomics) and counts the
// distinct experts executed.  Physical residency is handled by the fill
// kernel.
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
#include "combine.h"

namespace cmoe {

namespace {

constexpr int kPolicyRouter = 0, kPolicyLRU = 1, kPolicyLFU = 2;  // cmoe_policy; 3 = LRFU

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

// Cross-lane steps without the LDS crossbar (all 64 lanes active):
// DPP quad permutations and mirrors inside 16-lane rows, and the gfx950
// permlane swaps across rows.  permlane16_swap(x, x) returns, in every lane,
// the pair {own value, value of lane ^ 16} in some order (permlane32_swap:
// lane ^ 32), so an order-free combine of the pair is the combine with that
// partner.
// Lanes whose source is outside their row read 0 (bound_ctrl); no step
// below uses such a lane's result.  The move folds into the consuming
// max or add as one DPP instruction.
template <int CTRL>
__device__ inline unsigned dpp(unsigned v) {
    return (unsigned)__builtin_amdgcn_mov_dpp((int)v, CTRL, 0xF, 0xF, true);
}
constexpr int kQuadXor1 = 0xB1;     // quad_perm 1,0,3,2
constexpr int kQuadXor2 = 0x4E;     // quad_perm 2,3,0,1
constexpr int kRowHalfMirror = 0x141;
constexpr int kRowMirror = 0x140;
constexpr int kRowShl1 = 0x101;     // lane i reads lane i + n of its row

// maximum (MAX) or minimum of a 32-bit unsigned value over the wavefront,
// wave-uniform
template <bool MAX>
__device__ inline uint32_t wave_reduce_u32(uint32_t v) {
    auto op = [](uint32_t a, uint32_t b) { return MAX ? (a > b ? a : b) : (a < b ? a : b); };
    v = op(v, dpp<kQuadXor1>(v));
    v = op(v, dpp<kQuadXor2>(v));
    v = op(v, dpp<kRowHalfMirror>(v));
    v = op(v, dpp<kRowMirror>(v));
    const auto p = __builtin_amdgcn_permlane16_swap(v, v, false, false);
    v = op(p[0], p[1]);
    const auto q = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    v = op(q[0], q[1]);
    return __builtin_amdgcn_readfirstlane(v);
}

// The largest key (wave-uniform) and the lowest expert index e = 64 j + lane
// holding it: a 32-bit reduction, then one ballot per register.
template <int NPL>
__device__ inline int argmax_lowest(const uint32_t (&key)[NPL], uint32_t& kmax) {
    uint32_t b = key[0];
#pragma unroll
    for (int j = 1; j < NPL; ++j) b = key[j] > b ? key[j] : b;
    kmax = wave_reduce_u32<true>(b);
    int e = -1;
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
        const unsigned long long bal = __ballot(key[j] == kmax);
        if (e < 0 && bal) e = j * 64 + __builtin_ctzll(bal);
    }
    return e;
}

// The fixed softmax (described at the top of this file) of R independent
// logit vectors, step by step for all of them at once so that the latencies
// of their cross-lane reductions overlap.  Wavefront maximum: DPP and
// permlane-swap max steps; sum: strided halving over the next power of two
// P >= N, in-lane adds for w >= 64, then for w = 32 .. 1 lane i < w adds lane
// i + w (the tree of lane 0 is exactly that order), lane 0's total taken.
template <int NPL, int R>
__device__ inline void softmax_fixed(const float (&z)[3][NPL], int N, int lane, float (&p)[3][NPL]) {
    unsigned u[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        float m = -INFINITY;
#pragma unroll
        for (int j = 0; j < NPL; ++j)
            if (j * 64 + lane < N) m = fmaxf(m, z[r][j]);
        u[r] = __float_as_uint(m);
    }
    // wavefront maxima
#pragma unroll
    for (int r = 0; r < R; ++r) u[r] = __float_as_uint(fmaxf(__uint_as_float(u[r]), __uint_as_float(dpp<kQuadXor1>(u[r]))));
#pragma unroll
    for (int r = 0; r < R; ++r) u[r] = __float_as_uint(fmaxf(__uint_as_float(u[r]), __uint_as_float(dpp<kQuadXor2>(u[r]))));
#pragma unroll
    for (int r = 0; r < R; ++r)
        u[r] = __float_as_uint(fmaxf(__uint_as_float(u[r]), __uint_as_float(dpp<kRowHalfMirror>(u[r]))));
#pragma unroll
    for (int r = 0; r < R; ++r) u[r] = __float_as_uint(fmaxf(__uint_as_float(u[r]), __uint_as_float(dpp<kRowMirror>(u[r]))));
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const auto q = __builtin_amdgcn_permlane16_swap(u[r], u[r], false, false);
        u[r] = __float_as_uint(fmaxf(__uint_as_float(q[0]), __uint_as_float(q[1])));
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const auto q = __builtin_amdgcn_permlane32_swap(u[r], u[r], false, false);
        u[r] = __float_as_uint(fmaxf(__uint_as_float(q[0]), __uint_as_float(q[1])));
    }
    float v[R][NPL];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const float m = __uint_as_float(__builtin_amdgcn_readfirstlane(u[r]));
#pragma unroll
        for (int j = 0; j < NPL; ++j) {
            const bool in = j * 64 + lane < N;
            p[r][j] = in ? canon_exp(z[r][j] - m) : 0.0f;
            v[r][j] = p[r][j];
        }
    }
    int P = 1;
    while (P < N) P <<= 1;
#pragma unroll
    for (int jw = NPL / 2; jw >= 1; jw >>= 1) {
        if (jw * 64 * 2 <= P) {
#pragma unroll
            for (int r = 0; r < R; ++r)
#pragma unroll
                for (int j = 0; j < jw; ++j) v[r][j] = v[r][j] + v[r][j + jw];
        }
    }
    // cross-lane halving steps (w < 64)
    const int Pw = P < 64 ? P : 64;
    float x[R];
#pragma unroll
    for (int r = 0; r < R; ++r) x[r] = v[r][0];
    if (Pw >= 64) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const unsigned w = __float_as_uint(x[r]);
            const auto q = __builtin_amdgcn_permlane32_swap(w, w, false, false);
            x[r] = x[r] + __uint_as_float(q[1]);
        }
    }
    if (Pw >= 32) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const unsigned w = __float_as_uint(x[r]);
            const auto q = __builtin_amdgcn_permlane16_swap(w, w, false, false);
            x[r] = x[r] + __uint_as_float(q[1]);
        }
    }
    if (Pw >= 16) {
#pragma unroll
        for (int r = 0; r < R; ++r) x[r] = x[r] + __uint_as_float(dpp<kRowShl1 + 7>(__float_as_uint(x[r])));
    }
    if (Pw >= 8) {
#pragma unroll
        for (int r = 0; r < R; ++r) x[r] = x[r] + __uint_as_float(dpp<kRowShl1 + 3>(__float_as_uint(x[r])));
    }
    if (Pw >= 4) {
#pragma unroll
        for (int r = 0; r < R; ++r) x[r] = x[r] + __uint_as_float(dpp<kRowShl1 + 1>(__float_as_uint(x[r])));
    }
    if (Pw >= 2) {
#pragma unroll
        for (int r = 0; r < R; ++r) x[r] = x[r] + __uint_as_float(dpp<kRowShl1>(__float_as_uint(x[r])));
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const float sum = __uint_as_float(__builtin_amdgcn_readlane(__float_as_uint(x[r]), 0));
#pragma unroll
        for (int j = 0; j < NPL; ++j) p[r][j] = p[r][j] / sum;
    }
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
    uint32_t key[NPL];
    bool in[NPL];
    uint32_t b = 0xFFFFFFFFu;
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
        const int e = j * 64 + lane;
        in[j] = e < N && ((member[j] >> lane) & 1ull);
        key[j] = in[j] ? ord32(sc[j]) : 0xFFFFFFFFu;
        b = key[j] < b ? key[j] : b;
    }
    const uint32_t kmin = wave_reduce_u32<false>(b);
    int e = -1;
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
        const unsigned long long bal = __ballot(in[j] && key[j] == kmin);
        if (e < 0 && bal) e = j * 64 + __builtin_ctzll(bal);
    }
    return e < 0 ? ~0ull : (((unsigned long long)kmin << 32) | (unsigned)e);
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
__device__ void refine_one(const Layout& lo, int s, int rl, int R, int t, bool counted, const float (&pred)[NPL],
                           const float (&aTv)[NPL], const unsigned long long (&cw_in)[NPL], int64_t ctr_p, int lane) {
    const int N = lo.N;
    float sST[NPL];
    uint32_t cand[NPL];  // ordered scores; 0 = not a candidate (no real score maps to 0)
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
        const int e = j * 64 + lane;
        if (e < N) {
            sST[j] = aTv[j] + pred[j];
            cand[j] = ord32(sST[j]);
        } else {
            sST[j] = 0.0f;
            cand[j] = 0u;
        }
    }
    unsigned long long* cptr = lo.cache + ((int64_t)s * lo.L + rl) * lo.NW;
    unsigned long long cw[NPL];
    int count = 0;
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
        cw[j] = j < lo.NW ? cw_in[j] : 0ull;
        count += __popcll(cw[j]);
    }
    int nP = 0;
    unsigned long long ins[NPL];  // experts inserted here
#pragma unroll
    for (int j = 0; j < NPL; ++j) ins[j] = 0ull;
    const int Rn = R < N ? R : N;
    for (int i = 0; i < Rn; ++i) {
        uint32_t ord_e;
        const int e = argmax_lowest(cand, ord_e);  // highest s^ST, lower index on ties
#pragma unroll
        for (int j = 0; j < NPL; ++j)
            if (j == (e >> 6) && lane == (e & 63)) cand[j] = 0u;
        if (bit_of(cw, e)) continue;              // already resident
        if (count < lo.C) {
            set_bit(cw, e);
            set_bit(ins, e);
            ++count;
            ++nP;
        } else {
            const unsigned long long mn = argmin_member(sST, cw, N, lane);
            const int v = (int)(mn & 0xFFFFFFFFull);
            const uint32_t ord_v = (uint32_t)(mn >> 32);
            if (ord_e > ord_v) {  // strictly higher priority
                clear_bit(cw, v);
                clear_bit(ins, v);
                set_bit(cw, e);
                set_bit(ins, e);
                ++nP;
            }
        }
    }
    if (lo.policy == kPolicyLRU) {  // inserted as the most recently used, at 2t + 1
#pragma unroll
        for (int j = 0; j < NPL; ++j) {
            const int e = j * 64 + lane;
            if (e < N && ((ins[j] >> lane) & 1ull)) lo.pol[((int64_t)s * lo.L + rl) * N + e] = (float)(2 * t + 1);
        }
    }
    if (lane == 0) {
        for (int j = 0; j < lo.NW; ++j) cptr[j] = cw[j];
        lo.events[((int64_t)rl * lo.S + s) * 4 + 2] = nP;
        if (counted) lo.ctr[((int64_t)s * lo.L + rl) * kNctr + kCtrP] = ctr_p + nP;
    }
}

template <int NPL, int NR, bool INJECT, int ZS>
__device__ void stream_step(const Layout& lo, const StepArgs& a, int s, int lane) {
    const int N = lo.N, L = lo.L, K = lo.K;
    const bool spatio = lo.iS > 0;           // a Spatio Router: stores a-score and p^S
    const bool classical = lo.policy != kPolicyRouter;
    const bool counted = (a.flags & kFlagCount) != 0;
    float pred[NPL];

    // Loads that do not depend on this token's scores are issued first so
    // that their latencies overlap: the refined layer's a^T and cache words,
    // the accessed layer's cache words and classical priorities, and the
    // counters.  They are issued whatever the flags (rows clamped into range,
    // words and experts past the end masked where they are used): a load
    // under a branch of its own makes the compiler wait for it where the
    // branches join, before the router partials below are even requested.
    const bool refine = (a.flags & kFlagRefine) != 0;
    const int64_t row_a = (int64_t)s * L + a.l, row_r = (int64_t)s * L + min(a.rl, L - 1);
    float aTv[NPL], polv[NPL], pS_st[NPL];
    unsigned long long cw_r[NPL], cw_a[NPL];
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
        const int ec = min(j * 64 + lane, N - 1), jw = min(j, lo.NW - 1);
        pS_st[j] = lo.pS[(int64_t)s * N + ec];  // the stored prediction, for a refine-only launch
        aTv[j] = lo.aT[row_r * N + ec];
        cw_r[j] = lo.cache[row_r * lo.NW + jw];
        cw_a[j] = lo.cache[row_a * lo.NW + jw];
        polv[j] = lo.pol[row_a * N + ec];
    }
    // counters this wavefront updates (lane 0 owns them)
    int64_t ctr_a[kNctr];
#pragma unroll
    for (int c = 0; c < kNctr; ++c) ctr_a[c] = lo.ctr[row_a * kNctr + c];
    const int64_t ctr_rp = lo.ctr[row_r * kNctr + kCtrP];
    int64_t bucket = 0;  // lane k < K: bucket of its selection and position in it
    int bucket_pos = 0;

    if (a.flags & kFlagAccess) {
        const int l = a.l;
        const int64_t sl = (int64_t)s * L + l;
        // logits: every load is issued first (router split partials, ZS slots
        // per logit, or the injected logits; the native bias, a zero row when
        // there is none), then the splits are added in ascending order and
        // rounded once
        const float* brow = lo.bias ? lo.bias + (int64_t)l * N : lo.zero_row;
        double2 pv[NR][NPL][ZS / 2];
        float zin[NR][NPL], bz[NPL];
#pragma unroll
        for (int j = 0; j < NPL; ++j) {
            const int e = j * 64 + lane;
            const int ec = e < N ? e : N - 1;  // lanes past N read a valid address and discard it
            bz[j] = brow[ec];
#pragma unroll
            for (int r = 0; r < NR; ++r) {
                if (INJECT) {
                    zin[r][j] = a.z[r][sl * N + ec];
                } else {
                    const double2* zp =
                        reinterpret_cast<const double2*>(lo.zpart + (((int64_t)s * NR + r) * N + ec) * ZS);
#pragma unroll
                    for (int u = 0; u < ZS / 2; ++u) pv[r][j][u] = zp[u];
                }
            }
        }
        float z[3][NPL];
#pragma unroll
        for (int r = NR; r < 3; ++r)
#pragma unroll
            for (int j = 0; j < NPL; ++j) z[r][j] = 0.0f;
#pragma unroll
        for (int r = 0; r < NR; ++r) {
#pragma unroll
            for (int j = 0; j < NPL; ++j) {
                float v;
                if (INJECT) {
                    v = zin[r][j];
                } else {
                    double acc = 0.0;
#pragma unroll
                    for (int p = 0; p < ZS; ++p)
                        if (p < lo.nsplit) acc += (p & 1) ? pv[r][j][p >> 1].y : pv[r][j][p >> 1].x;
                    if (r == 0) acc += (double)bz[j];
                    v = (float)acc;
                }
                const int e = j * 64 + lane;
                if (e < N) lo.logits[(((int64_t)l * lo.S + s) * NR + r) * N + e] = v;
                z[r][j] = e < N ? v : 0.0f;
            }
        }
        // router slots: 0 native, then temporal (router policy), then spatio;
        // every slot is in use, so the NR softmaxes run together
        float pz[3][NPL];
        softmax_fixed<NPL, NR>(z, N, lane, pz);
        float pR[NPL], pT[NPL];
#pragma unroll
        for (int j = 0; j < NPL; ++j) {
            pR[j] = pz[0][j];
            pT[j] = (NR >= 2 && !classical) ? pz[1][j] : 0.0f;
            if (NR >= 2 && spatio) pred[j] = pz[NR - 1][j];
        }

        // Top-K by native logit, lower index first on ties
        uint32_t key[NPL];  // ordered native logits; 0 = taken or past N (no real logit maps to 0)
#pragma unroll
        for (int j = 0; j < NPL; ++j) {
            const int e = j * 64 + lane;
            key[j] = e < N ? ord32(z[0][j]) : 0u;
        }
        unsigned long long sw[NPL];
#pragma unroll
        for (int j = 0; j < NPL; ++j) sw[j] = 0ull;
        float gsum = 0.0f, my_p = 0.0f;
        int my_sel = 0;
        for (int k = 0; k < K; ++k) {
            uint32_t kmax;
            const int e = argmax_lowest(key, kmax);  // highest logit, lower index on ties
            float pv = 0.0f;
#pragma unroll
            for (int j = 0; j < NPL; ++j) {
                if (j == (e >> 6) && lane == (e & 63)) {
                    key[j] = 0u;
                    pv = pR[j];
                }
            }
            pv = __uint_as_float(__builtin_amdgcn_readlane(__float_as_uint(pv), e & 63));
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
            // token (s, k) joins the bucket of its expert; the position inside
            // the bucket does not affect any result (each token is its own
            // column of the expert's matrix products).  The position is used
            // at the end of the step, so the atomic's round trip overlaps the
            // rest of it.
            bucket = (int64_t)a.bbuf * N + my_sel;
            bucket_pos = atomicAdd(&lo.bcount[bucket], 1);
            if (counted) atomicAdd(&lo.selcount[(int64_t)l * N + my_sel], 1ull);
        }
        // retention priority of Algorithm 1
        float sT[NPL];
        if (!classical) {
#pragma unroll
            for (int j = 0; j < NPL; ++j) sT[j] = pR[j] + pT[j];
        } else {
#pragma unroll
            for (int j = 0; j < NPL; ++j) {
                const bool used = (sw[j] >> lane) & 1ull;
                float v = j * 64 + lane < N ? polv[j] : 0.0f;
                if (lo.policy == kPolicyLRU) {
                    if (used) v = (float)(2 * a.t + 2);
                } else if (lo.policy == kPolicyLFU) {
                    if (used) v = v + 1.0f;
                } else {
                    v = v * lo.lrfu_w;
                    if (used) v = v + 1.0f;
                }
                sT[j] = v;
                const int e = j * 64 + lane;
                if (e < N) lo.pol[sl * N + e] = v;
            }
        }

        // access
        unsigned long long* cptr = lo.cache + sl * lo.NW;
        unsigned long long cw[NPL];
        int count = 0, hits = 0;
#pragma unroll
        for (int j = 0; j < NPL; ++j) {
            cw[j] = j < lo.NW ? cw_a[j] : 0ull;
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
            for (int j = 0; j < lo.NW; ++j) cptr[j] = cw[j];
            int32_t* ev = lo.events + ((int64_t)l * lo.S + s) * 4;
            ev[0] = hits;
            ev[1] = nD;
            if (!(a.flags & kFlagRefinedHere)) ev[2] = 0;
            ev[3] = 0;
            if (counted) {
                int64_t* c = lo.ctr + sl * kNctr;
                c[kCtrA] = ctr_a[kCtrA] + K;
                c[kCtrHits] = ctr_a[kCtrHits] + hits;
                c[kCtrD] = ctr_a[kCtrD] + nD;
                c[kCtrT] = ctr_a[kCtrT] + 1;
            }
        }
        if (spatio) {  // the next token's a-score of this layer, and p^S for the successor
            const bool spatio_only = lo.iT < 0;
#pragma unroll
            for (int j = 0; j < NPL; ++j) {
                const int e = j * 64 + lane;
                if (e < N) {
                    lo.aT[sl * N + e] = spatio_only ? pR[j] : sT[j];
                    lo.pS[(int64_t)s * N + e] = pred[j];
                }
            }
        }
        // The refinement is called on each side of the branch: after a join
        // with the refine-only side, whose prediction loads may still be in
        // flight there, the compiler waits for every outstanding memory
        // operation, and with it for the bucket atomic issued above, whose
        // round trip the refinement is meant to hide.
        if (refine) refine_one<NPL>(lo, s, a.rl, a.R, a.t, counted, pred, aTv, cw_r, ctr_rp, lane);
    } else {
        // refine-only launch: the predecessor's prediction is the stored one
#pragma unroll
        for (int j = 0; j < NPL; ++j) {
            const int e = j * 64 + lane;
            pred[j] = e < N ? pS_st[j] : 0.0f;
        }
        if (refine) refine_one<NPL>(lo, s, a.rl, a.R, a.t, counted, pred, aTv, cw_r, ctr_rp, lane);
    }
    if ((a.flags & kFlagAccess) && lane < K) {
        lo.pairs[bucket * lo.S + bucket_pos] = (s << 8) | lane;
        if (counted && bucket_pos == 0) atomicAdd(&lo.active_sum[a.l], 1ull);
    }
}

// grid: the stream workgroups, then (a.y non-NULL) the workgroups of the
// previous layer's combine.  The combine's only input, the gated expert
// outputs, is complete once the previous layer's FFN has run, and no step of
// this launch reads its output, so it runs here on the compute units that the
// stream wavefronts leave idle, in place of a launch of its own; its
// workgroups come after the streams' in dispatch order, so the streams'
// prologue loads are issued first.
template <int NPL, int NR, bool INJECT, int ZS>
__global__ __launch_bounds__(64 * kStreamsPerBlock) void cache_step_kernel(Layout lo, StepArgs a) {
    constexpr int kThreads = 64 * kStreamsPerBlock;
    const int nsb = (lo.S + kStreamsPerBlock - 1) / kStreamsPerBlock;
    if ((int)blockIdx.x >= nsb) {
        combine_quad(lo, a.cl, a.y, (int64_t)(blockIdx.x - nsb) * kThreads + threadIdx.x);
        return;
    }
    const int lane = threadIdx.x & 63;
    const int s = blockIdx.x * kStreamsPerBlock + (threadIdx.x >> 6);
    if ((a.flags & kFlagAccess) && blockIdx.x == 0) {
        // the other bucket buffer was used by the previous layer step (its FFN
        // has completed) and is filled by the next one
        for (int i = threadIdx.x; i < lo.N; i += kThreads) lo.bcount[(int64_t)(a.bbuf ^ 1) * lo.N + i] = 0;
    }
    if (s < lo.S) stream_step<NPL, NR, INJECT, ZS>(lo, a, s, lane);  // wave-uniform branch
}

// ---------------------------------------------------------------- init
__global__ void init_kernel(Layout lo) {
    const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t gs = (int64_t)gridDim.x * blockDim.x;
    const int64_t nc = (int64_t)lo.S * lo.L * lo.NW;
    for (int64_t i = gid; i < nc; i += gs) lo.cache[i] = 0ull;
    const int64_t na = (int64_t)lo.S * lo.L * lo.N;
    for (int64_t i = gid; i < na; i += gs) {
        lo.aT[i] = 0.0f;
        lo.pol[i] = 0.0f;
    }
    for (int64_t i = gid; i < (int64_t)lo.S * lo.N; i += gs) lo.pS[i] = 0.0f;
    for (int64_t i = gid; i < (int64_t)lo.S * lo.L * kNctr; i += gs) lo.ctr[i] = 0;
    for (int64_t i = gid; i < (int64_t)lo.L * 2; i += gs) lo.phys[i] = 0;
    for (int64_t i = gid; i < lo.L; i += gs) lo.active_sum[i] = 0ull;
    for (int64_t i = gid; i < (int64_t)lo.L * lo.N; i += gs) lo.selcount[i] = 0ull;
    for (int64_t i = gid; i < (int64_t)2 * lo.L * lo.N; i += gs) lo.slot_of[i] = -1;
    for (int64_t i = gid; i < (int64_t)2 * lo.L * lo.n_slots; i += gs) {
        lo.slot_exp[i] = -1;
        lo.slot_stamp[i] = 0;
    }
    if (lo.events == nullptr) return;  // no workspace bound (kernel-uniform)
    for (int64_t i = gid; i < (int64_t)lo.L * 2; i += gs) lo.step_fills[i] = 0;
    for (int64_t i = gid; i < (int64_t)lo.L * lo.S * 4; i += gs) lo.events[i] = 0;
    for (int64_t i = gid; i < (int64_t)2 * lo.N; i += gs) lo.bcount[i] = 0;
    for (int64_t i = gid; i < lo.N; i += gs) lo.zero_row[i] = 0.0f;
}

// What a token's first layer step needs zero in a workspace that other calls
// may have left behind: both bucket-count buffers and the zero bias row.
__global__ __launch_bounds__(256) void prep_workspace_kernel(Layout lo) {
    for (int i = threadIdx.x; i < 2 * lo.N; i += blockDim.x) lo.bcount[i] = 0;
    for (int i = threadIdx.x; i < lo.N; i += blockDim.x) lo.zero_row[i] = 0.0f;
}

}  // namespace

hipError_t launch_init(const Layout& lo, hipStream_t st) {
    hipLaunchKernelGGL(init_kernel, dim3(256), dim3(256), 0, st, lo);
    return hipGetLastError();
}

hipError_t launch_prep_workspace(const Layout& lo, hipStream_t st) {
    hipLaunchKernelGGL(prep_workspace_kernel, dim3(1), dim3(256), 0, st, lo);
    return hipGetLastError();
}

template <int NPL, int NR>
hipError_t launch_step_nr(const Layout& lo, const StepArgs& a, hipStream_t st, const Timing& tm) {
    const int64_t nsb = (lo.S + kStreamsPerBlock - 1) / kStreamsPerBlock;
    const int64_t quads = a.y ? (int64_t)lo.S * (lo.d / 4) : 0;  // combine threads
    const dim3 grid((unsigned)(nsb + (quads + 64 * kStreamsPerBlock - 1) / (64 * kStreamsPerBlock)));
    const dim3 block(64 * kStreamsPerBlock);
    if (a.flags & kFlagInject)
        launch_kernel(cache_step_kernel<NPL, NR, true, 2>, grid, block, st, tm, lo, a);
    else if (lo.zstride == 4)
        launch_kernel(cache_step_kernel<NPL, NR, false, 4>, grid, block, st, tm, lo, a);
    else
        launch_kernel(cache_step_kernel<NPL, NR, false, kMaxSplit>, grid, block, st, tm, lo, a);
    return hipGetLastError();
}

template <int NPL>
hipError_t launch_step_npl(const Layout& lo, const StepArgs& a, hipStream_t st, const Timing& tm) {
    if (lo.n_r == 3) return launch_step_nr<NPL, 3>(lo, a, st, tm);
    if (lo.n_r == 2) return launch_step_nr<NPL, 2>(lo, a, st, tm);
    return launch_step_nr<NPL, 1>(lo, a, st, tm);
}

hipError_t launch_cache_step(const Layout& lo, const StepArgs& a, hipStream_t st, const Timing& tm) {
    if (lo.N <= 64) return launch_step_npl<1>(lo, a, st, tm);
    if (lo.N <= 128) return launch_step_npl<2>(lo, a, st, tm);
    return launch_step_npl<4>(lo, a, st, tm);
}

}  // namespace cmoe
