/*
 * oracle.c - plain, slow CPU oracle of the cache-aware MoE decode step.
 *
 * TEST INFRASTRUCTURE.  Only the tests, the smoke check and the benchmark's
 * CPU-baseline leg load this library; the product path never does.  It shares
 * no code with the GPU path.
 *
 * What it computes, and where the paper defines it:
 *   - native router p^R = softmax(W^R h), S = TopK(p^R)          (Section 2)
 *   - Temporal Router p^T = softmax(W^T h), s^T = p^R + p^T      (Section 3.2)
 *   - post-access retention U_B, the shared cache update        (Algorithm 1)
 *   - Spatio Router p^S = softmax(W^S h), causal predecessor rho,
 *     a^T = p^R_{t-1} + p^T_{t-1}, s^ST = a^T + p^S_rho            (Section 3.3)
 *   - pre-access refinement over Top_R(s^ST)                      (Algorithm 2,
 *     Section 3.3 last paragraph, Appendix B.2)
 *   - accounting A, D, P, T and Hit, AdjHit, Load/token           (Section 4.1
 *     "Metrics")
 *   - the classical cache-update baselines LRU, LFU and LRFU (Section 4.1
 *     baselines, Table 1 "Cache-Update Methods", LRFU with lambda = 0.5),
 *     written from their textbook definitions (Mattson et al. 1970 for
 *     recency; frequency counts; Lee et al. 2001 for the combined
 *     recency-frequency value with weighing function (1/2)^(lambda x)), as
 *     the retention priority of the same post-access update (Algorithm 1)
 *   - expert-use concentration of the native selections (Section 5,
 *     "routing behaviour" figure): per layer the selection frequencies f_e
 *     (normalised to sum 1), effective experts exp(H), entropy H in nats,
 *     max frequency and top-m mass, averaged over layers
 *   - the Spatio-only ablation (Section 5 ablations, Appendix B.4):
 *     s^S = p^R_{t-1,l} + p^S_rho drives the pre-access refinement, and
 *     demand-miss insertion evicts by LRU
 *   - SwiGLU expert FFN on the selected experts ("execute the MoE layer",
 *     Algorithm 2), in fp64.
 *
 * Readings where the paper is silent (each listed in the design notes):
 *   - Scores use a fixed fp32 arithmetic, "canonical" below, so that a second
 *     implementation can reproduce every comparison bit for bit: logits are
 *     summed in fp64 and rounded once to fp32; softmax uses orc_exp (Cody-Waite
 *     reduction + degree-7 Taylor polynomial), a strided-halving sum and an
 *     IEEE division; score sums are single fp32 additions.
 *   - Top-K ranks the fp32 native logits (softmax is monotone); all ties go to
 *     the lower expert index, argmin ties evict the lower index, replacement
 *     during refinement needs a strictly higher score.
 *   - Demand-loaded experts are inserted in ascending index order.
 *   - Caches start empty; refinement starts at the second token.
 *   - Gate weights are the selected native probabilities renormalised to 1.
 *   - Physical residency: per layer the device holds the union of the streams'
 *     caches in numbered slots; a newly needed expert takes the lowest free
 *     slot, in ascending expert order.  Refinement and the post-access update
 *     each end with such a residency event.
 *   - A capacity-limited arena (fewer slots per layer than the union of the
 *     caches can reach, the paper's bounded device cache taken literally for
 *     many streams) is a second-level cache over the slots: when the union
 *     fits it behaves as above; when it does not, the layer step's executed
 *     experts pass through the slots in rounds of at most n_slots experts
 *     (the experts already resident first, then the others, each group in
 *     ascending order), every missing expert taking the lowest free slot or
 *     else evicting the least recently used expert that no remaining round
 *     needs (lower slot on equal recency), and refinement only fills free
 *     slots.
 *   - Classical priorities live per (stream, layer, expert) and are updated
 *     once per access, before the eviction decision: LRU stores the time of
 *     the last use (0 = never), LFU the number of selections, LRFU
 *     C <- fl32(C * w) (+ 1 if selected), w = fl32(2^-lambda), for every
 *     expert.  LRU time counts two events per token t: the pre-access
 *     refinement at 2t + 1 and the access at 2t + 2.  An expert inserted
 *     proactively (Spatio-only mode) takes time 2t + 1, i.e. enters as the
 *     most recently used, behind the experts selected at the access that
 *     follows; frequency policies do not count an insertion as a use.
 *
 * Build: gcc -O2 -ffp-contract=off (no fused multiply-add contraction, no
 * fast-math); fmaf/rintf/ldexpf are the C library's correctly rounded ones.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_NMAX 1024

/* ------------------------------------------------------------------ */
/* Canonical fp32 exponential for x <= 0.                              */
/* ------------------------------------------------------------------ */
/* ln 2 split (Cody & Waite): the high part keeps the top bits of fl32(ln 2)
 * with the low 8 bits of its 23-bit fraction cleared, so k*LN2_HI is exact
 * for |k| < 2^8; the low part is fl32(ln 2 - LN2_HI). */
static float g_ln2_hi, g_ln2_lo, g_inv_ln2, g_coef[8];
static int g_init = 0;

static void orc_init_constants(void) {
    if (g_init) return;
    double ln2 = log(2.0);
    float f = (float)ln2;
    uint32_t u;
    memcpy(&u, &f, 4);
    u &= ~(uint32_t)0xFF;
    memcpy(&g_ln2_hi, &u, 4);
    g_ln2_lo = (float)(ln2 - (double)g_ln2_hi);
    g_inv_ln2 = (float)(1.0 / ln2);
    double fact = 1.0;
    for (int n = 0; n < 8; ++n) {
        if (n > 0) fact *= (double)n;
        g_coef[n] = (float)(1.0 / fact); /* Taylor coefficients 1/n! */
    }
    g_init = 1;
}

void orc_exp_constants(float* out /* [11]: ln2_hi, ln2_lo, inv_ln2, c0..c7 */) {
    orc_init_constants();
    out[0] = g_ln2_hi;
    out[1] = g_ln2_lo;
    out[2] = g_inv_ln2;
    for (int n = 0; n < 8; ++n) out[3 + n] = g_coef[n];
}

float orc_exp(float x) {
    orc_init_constants();
    if (x < -80.0f) return 0.0f;
    float k = rintf(x * g_inv_ln2);           /* nearest integer, ties to even */
    float r = fmaf(-k, g_ln2_hi, x);          /* exact: x - k*ln2_hi */
    r = fmaf(-k, g_ln2_lo, r);
    float p = g_coef[7];
    for (int n = 6; n >= 0; --n) p = fmaf(p, r, g_coef[n]);   /* Horner */
    return ldexpf(p, (int)k);
}

/* Canonical softmax: m = max z; u = exp(z - m); sum by strided halving over
 * the next power of two (padding with +0): v[i] += v[i + w] for w = P/2 .. 1;
 * p = u / sum. */
void orc_softmax(const float* z, int n, float* p) {
    float m = z[0];
    for (int e = 1; e < n; ++e)
        if (z[e] > m) m = z[e];
    int P = 1;
    while (P < n) P <<= 1;
    float v[ORC_NMAX];
    for (int e = 0; e < P; ++e) v[e] = 0.0f;
    for (int e = 0; e < n; ++e) {
        float diff = z[e] - m;
        p[e] = orc_exp(diff);
        v[e] = p[e];
    }
    for (int w = P / 2; w >= 1; w /= 2)
        for (int i = 0; i < w; ++i) v[i] = v[i] + v[i + w];
    for (int e = 0; e < n; ++e) p[e] = p[e] / v[0];
}

/* ------------------------------------------------------------------ */
/* Ranking                                                             */
/* ------------------------------------------------------------------ */
/* The k largest entries of v in descending order; equal values: lower index
 * first.  (-0 and +0 compare equal, so they tie.) */
void orc_topk(const float* v, int n, int k, int32_t* out) {
    uint8_t taken[ORC_NMAX];
    memset(taken, 0, (size_t)n);
    for (int r = 0; r < k; ++r) {
        int best = -1;
        for (int e = 0; e < n; ++e) {
            if (taken[e]) continue;
            if (best < 0 || v[e] > v[best]) best = e;
        }
        taken[best] = 1;
        out[r] = best;
    }
}

/* The (up to) k members of `allowed` with the lowest scores, lowest first;
 * equal scores: lower index first.  Returns how many there are. */
static int orc_lowest(const float* s, const uint8_t* allowed, int n, int k, int32_t* out) {
    uint8_t taken[ORC_NMAX];
    memset(taken, 0, (size_t)n);
    int found = 0;
    while (found < k) {
        int best = -1;
        for (int u = 0; u < n; ++u)
            if (allowed[u] && !taken[u] && (best < 0 || s[u] < s[best])) best = u;
        if (best < 0) break;
        taken[best] = 1;
        out[found++] = best;
    }
    return found;
}

static int orc_count(const uint8_t* c, int n) {
    int k = 0;
    for (int e = 0; e < n; ++e) k += c[e] ? 1 : 0;
    return k;
}

/* ------------------------------------------------------------------ */
/* Post-access retention U_B(C, S, s) (Section 3.2, Algorithm 1)        */
/* ------------------------------------------------------------------ */
/* After the access every selected expert is resident: the demand misses
 * D = S \ C are loaded, and nothing else is admitted.  When C u S exceeds
 * the capacity, the surplus leaves: the residents outside S with the lowest
 * priority, lower index first among equal priorities (the residents that
 * Algorithm 1 evicts one demand at a time, since S is protected and the
 * candidates for eviction only shrink).
 * C: membership [N] (0/1), updated in place.  S: the K selected experts.
 * s: retention priority (s^T).  demand (may be NULL): receives D in
 * ascending order.  Returns |D|. */
int orc_update_cache(uint8_t* C, int N, int cap, const int32_t* S, int K, const float* s,
                     int32_t* demand) {
    uint8_t sel[ORC_NMAX], leavable[ORC_NMAX];
    memset(sel, 0, (size_t)N);
    for (int k = 0; k < K; ++k) sel[S[k]] = 1;
    int32_t D[ORC_NMAX];
    int nD = 0;
    for (int e = 0; e < N; ++e)
        if (sel[e] && !C[e]) D[nD++] = e;
    const int surplus = orc_count(C, N) + nD - cap;
    if (surplus > 0) {
        for (int u = 0; u < N; ++u) leavable[u] = (uint8_t)(C[u] && !sel[u]);
        int32_t out[ORC_NMAX];
        const int n = orc_lowest(s, leavable, N, surplus, out);
        for (int i = 0; i < n; ++i) C[out[i]] = 0;
    }
    for (int i = 0; i < nD; ++i) C[D[i]] = 1;
    if (demand)
        for (int i = 0; i < nD; ++i) demand[i] = D[i];
    return nD;
}

/* ------------------------------------------------------------------ */
/* Pre-access refinement (Section 3.3, Algorithm 2)                     */
/* ------------------------------------------------------------------ */
/* The candidates A = Top_R(s^ST) are examined from the highest score down.
 * A candidate already resident stays; one that is not is loaded while the
 * cache has room, and after that displaces the weakest resident only when
 * its score is strictly higher.  Candidates come in non-increasing score and
 * the weakest remaining resident never gets weaker, so the displaced experts
 * are the weakest residents in order (lower index first among equals), and
 * the displacements stop at the first candidate that does not beat the next
 * of them.
 * C updated in place; loaded (may be NULL) receives the proactively loaded
 * experts in the order they are examined.  Returns their number. */
int orc_refine(uint8_t* C, int N, int cap, const float* sST, int R, int32_t* loaded) {
    int32_t A[ORC_NMAX], fresh[ORC_NMAX], weakest[ORC_NMAX];
    if (R > N) R = N;
    orc_topk(sST, N, R, A);
    int nfresh = 0;
    for (int i = 0; i < R; ++i)
        if (!C[A[i]]) fresh[nfresh++] = A[i];
    const int room = cap - orc_count(C, N);
    const int nfill = nfresh < room ? nfresh : room;
    for (int i = 0; i < nfill; ++i) C[fresh[i]] = 1;
    const int32_t* rest = fresh + nfill;
    const int nrest = nfresh - nfill;
    int nrep = 0;
    if (nrest > 0) {
        const int nw = orc_lowest(sST, C, N, nrest, weakest);
        while (nrep < nrest && nrep < nw && sST[rest[nrep]] > sST[weakest[nrep]]) ++nrep;
        for (int i = 0; i < nrep; ++i) {
            C[weakest[i]] = 0;
            C[rest[i]] = 1;
        }
    }
    if (loaded)
        for (int i = 0; i < nfill + nrep; ++i) loaded[i] = fresh[i];
    return nfill + nrep;
}

/* ------------------------------------------------------------------ */
/* Router logits and the expert FFN (textbook definitions, fp64)       */
/* ------------------------------------------------------------------ */
/* z_e = fl32( sum_i W[e][i] * h[i] + bias[e] ), accumulated in fp64. */
void orc_logits(const float* W, const float* h, const float* bias, int N, int d, float* z) {
    for (int e = 0; e < N; ++e) {
        double acc = 0.0;
        const float* w = W + (size_t)e * d;
        for (int i = 0; i < d; ++i) acc += (double)w[i] * (double)h[i];
        if (bias) acc += (double)bias[e];
        z[e] = (float)acc;
    }
}

/* y = sum_k g_k * W_down,k ( silu(W_gate,k x) * (W_up,k x) ), fp64.
 * Wg, Wu: [K][F][d]; Wd: [K][d][F]; silu(a) = a / (1 + exp(-a)). */
void orc_moe_ffn(const float* Wg, const float* Wu, const float* Wd, const double* g, int K, const float* x,
                 int d, int F, double* y) {
    double* act = (double*)malloc(sizeof(double) * (size_t)F);
    for (int j = 0; j < d; ++j) y[j] = 0.0;
    for (int k = 0; k < K; ++k) {
        const float* wg = Wg + (size_t)k * F * d;
        const float* wu = Wu + (size_t)k * F * d;
        const float* wd = Wd + (size_t)k * d * F;
        for (int f = 0; f < F; ++f) {
            double a = 0.0, b = 0.0;
            for (int i = 0; i < d; ++i) {
                a += (double)wg[(size_t)f * d + i] * (double)x[i];
                b += (double)wu[(size_t)f * d + i] * (double)x[i];
            }
            act[f] = a / (1.0 + exp(-a)) * b;
        }
        for (int j = 0; j < d; ++j) {
            double acc = 0.0;
            for (int f = 0; f < F; ++f) acc += (double)wd[(size_t)j * F + f] * act[f];
            y[j] += g[k] * acc;
        }
    }
    free(act);
}

/* Expert-use concentration from per-(layer, expert) selection counts
 * [L][N]: for each layer with at least one selection, f_e = count_e / sum,
 * H = -sum_{f_e > 0} f_e ln f_e, and out4 = the means over those layers of
 * exp(H), H, max_e f_e and the sum of the top_m largest f_e.  Returns the
 * number of layers averaged. */
int orc_concentration(const int64_t* counts, int L, int N, int top_m, double* out4) {
    double acc[4] = {0.0, 0.0, 0.0, 0.0};
    int used = 0;
    for (int l = 0; l < L; ++l) {
        const int64_t* c = counts + (size_t)l * N;
        int64_t tot = 0;
        for (int e = 0; e < N; ++e) tot += c[e];
        if (tot == 0) continue;
        double f[ORC_NMAX], H = 0.0, fmax = 0.0;
        for (int e = 0; e < N; ++e) {
            f[e] = (double)c[e] / (double)tot;
            if (f[e] > 0.0) H -= f[e] * log(f[e]);
            if (f[e] > fmax) fmax = f[e];
        }
        /* top-m mass: repeatedly take the largest remaining frequency */
        uint8_t taken[ORC_NMAX];
        memset(taken, 0, (size_t)N);
        double mass = 0.0;
        for (int i = 0; i < top_m && i < N; ++i) {
            int best = -1;
            for (int e = 0; e < N; ++e)
                if (!taken[e] && (best < 0 || f[e] > f[best])) best = e;
            taken[best] = 1;
            mass += f[best];
        }
        acc[0] += exp(H);
        acc[1] += H;
        acc[2] += fmax;
        acc[3] += mass;
        ++used;
    }
    for (int i = 0; i < 4; ++i) out4[i] = used ? acc[i] / used : 0.0;
    return used;
}

/* Hit = 1 - D/A, AdjHit = (A - D)/(A + P), Load/token = (D + P) S_exp / T in
 * decimal MB (Section 4.1 "Metrics"). */
void orc_metrics(int64_t A, int64_t D, int64_t P, int64_t T, double expert_bytes, double* out3) {
    out3[0] = 1.0 - (double)D / (double)A;
    out3[1] = (double)(A - D) / (double)(A + P);
    out3[2] = (double)(D + P) * expert_bytes / 1e6 / (double)T;
}

/* ------------------------------------------------------------------ */
/* One decode token for all streams                                    */
/* ------------------------------------------------------------------ */
enum { ORC_MODE_TEMPORAL = 0, ORC_MODE_SPATIO_TEMPORAL = 1, ORC_MODE_SPATIO_ONLY = 2 };
enum { ORC_POLICY_ROUTER = 0, ORC_POLICY_LRU = 1, ORC_POLICY_LFU = 2, ORC_POLICY_LRFU = 3 };

typedef struct {
    int32_t L, N, K, C, R, S, mode, warmup_tokens;
    int32_t policy;   /* retention priority of Algorithm 1: s^T or a classical one */
    float lrfu_w;     /* LRFU decay per token, fl32(2^-lambda)                    */
} orc_cfg;

enum { ORC_CTR_A = 0, ORC_CTR_HITS, ORC_CTR_D, ORC_CTR_P, ORC_CTR_T, ORC_NCTR };

typedef struct {
    uint8_t* cache;   /* [S][L][N] logical cache membership                    */
    float* aT;        /* [S][L][N] previous token's a-score: s^T (full mode),
                                    p^R (Spatio-only mode)                     */
    float* pS;        /* [S][N]    latest Spatio Router distribution           */
    int64_t* ctr;     /* [S][L][5] A, hits, D, P, T (counted tokens only)       */
    int32_t* slot_of; /* [L][N]    physical slot of each expert, -1 = absent   */
    int64_t* phys;    /* [L][2]    physical fills: demand, proactive (counted)  */
    float* pol;       /* [S][L][N] classical retention priority (policy != 0)  */
    int64_t* selcount;/* [L][N]    native selections per expert (counted tokens) */
    int64_t* stamp;   /* [L][N]    physical recency: the arena clock at the last
                                    use of each expert's copy (valid while resident) */
    int64_t* clk;     /* [L]       arena clock: advances once per round of a
                                    residency event                              */
    int32_t n_slots;  /* physical slots per layer                              */
    int32_t t;        /* index of the next token                               */
} orc_state;

typedef struct {      /* optional per-token outputs (any pointer may be NULL) */
    int32_t* sel;     /* [S][L][K] selected experts, descending native logit   */
    double* gate;     /* [S][L][K] renormalised selected probabilities         */
    float* pR;        /* [S][L][N] */
    float* sT;        /* [S][L][N] retention priority used by Algorithm 1      */
    float* sST;       /* [S][L][N] (full mode, t >= 1)                          */
    int32_t* hits;    /* [S][L] */
    int32_t* nD;      /* [S][L] */
    int32_t* nP;      /* [S][L] */
    int32_t* fills;   /* [L][2] physical fills of this token: demand, proactive */
} orc_out;

/* Lowest free slot of a layer's arena, or -1 when every slot is taken. */
static int orc_free_slot(const orc_state* st, int N, const int32_t* slot) {
    for (int q = 0; q < st->n_slots; ++q) {
        int used = 0;
        for (int u = 0; u < N; ++u)
            if (slot[u] == q) used = 1;
        if (!used) return q;
    }
    return -1;
}

/* Residency event of layer l.  U is the union of the streams' caches;
 * experts that left U free their slots.  E: the experts the layer step's FFN
 * executes (after the post-access update), or NULL (after refinement).
 *   - U fits the slots: every member of U becomes resident, each new one, in
 *     ascending order, in the lowest free slot.
 *   - U does not fit, after refinement: new members of U, in ascending order,
 *     take free slots while there are any.
 *   - U does not fit, after the post-access update: E is ordered, resident
 *     experts first, then the others, each group ascending, and executed in
 *     rounds of n_slots consecutive experts.  In its round each missing
 *     expert, in that order, takes the lowest free slot, or else the slot of
 *     the resident expert that no remaining round needs with the oldest last
 *     use (lower slot on ties), which is evicted.
 * The clock advances once per round (once in the first two cases); every
 * expert copied, and every expert executed in a round, gets it as its last
 * use.  Returns the number of copies. */
static int orc_residency(const orc_cfg* c, orc_state* st, int l, const uint8_t* E) {
    const int N = c->N;
    uint8_t inU[ORC_NMAX];
    memset(inU, 0, (size_t)N);
    for (int s = 0; s < c->S; ++s) {
        const uint8_t* cs = st->cache + ((size_t)s * c->L + l) * N;
        for (int e = 0; e < N; ++e)
            if (cs[e]) inU[e] = 1;
    }
    int32_t* slot = st->slot_of + (size_t)l * N;
    int64_t* stamp = st->stamp + (size_t)l * N;
    for (int e = 0; e < N; ++e)
        if (slot[e] >= 0 && !inU[e]) slot[e] = -1;
    const int nU = orc_count(inU, N);
    int fills = 0;
    if (nU <= st->n_slots || !E) {
        const int64_t now = ++st->clk[l];
        for (int e = 0; e < N; ++e) {
            if (!inU[e] || slot[e] >= 0) continue;
            const int q = orc_free_slot(st, N, slot);
            if (q < 0) {
                if (nU <= st->n_slots) return -1; /* cannot happen: the union fits */
                break;                            /* refinement: no free slot left */
            }
            slot[e] = q;
            stamp[e] = now;
            ++fills;
        }
        if (E)
            for (int e = 0; e < N; ++e)
                if (E[e]) stamp[e] = now;
        return fills;
    }
    int32_t order[ORC_NMAX], round_of[ORC_NMAX];
    int nE = 0;
    for (int e = 0; e < N; ++e)
        if (E[e] && slot[e] >= 0) order[nE++] = e;
    for (int e = 0; e < N; ++e)
        if (E[e] && slot[e] < 0) order[nE++] = e;
    for (int e = 0; e < N; ++e) round_of[e] = -1;
    for (int i = 0; i < nE; ++i) round_of[order[i]] = i / st->n_slots;
    for (int r = 0; r * st->n_slots < nE; ++r) {
        const int64_t now = ++st->clk[l];
        const int lo = r * st->n_slots, hi = lo + st->n_slots < nE ? lo + st->n_slots : nE;
        for (int i = lo; i < hi; ++i) {
            const int e = order[i];
            if (slot[e] >= 0) continue;
            int q = orc_free_slot(st, N, slot);
            if (q < 0) {
                int victim = -1;
                for (int v = 0; v < N; ++v) {
                    if (slot[v] < 0 || round_of[v] >= r) continue; /* absent, or needed now or later */
                    if (victim < 0 || stamp[v] < stamp[victim] ||
                        (stamp[v] == stamp[victim] && slot[v] < slot[victim]))
                        victim = v;
                }
                if (victim < 0) return -1; /* cannot happen: a round fits the slots */
                q = slot[victim];
                slot[victim] = -1;
            }
            slot[e] = q;
            ++fills;
        }
        for (int i = lo; i < hi; ++i) stamp[order[i]] = now;
    }
    return fills;
}

/* LRFU decay per token: the weighing function (1/2)^(lambda x) at x = 1,
 * rounded once to fp32. */
float orc_lrfu_weight(float lambda) { return (float)pow(2.0, -(double)lambda); }

/* Classical retention priority of one (stream, layer) at an access of token
 * t: the selected experts are used now. */
static void orc_policy_access(int policy, float w, float* pol, int N, const uint8_t* selected, int t) {
    for (int e = 0; e < N; ++e) {
        if (policy == ORC_POLICY_LRU) {
            if (selected[e]) pol[e] = (float)(2 * t + 2);
        } else if (policy == ORC_POLICY_LFU) {
            if (selected[e]) pol[e] = pol[e] + 1.0f;
        } else if (policy == ORC_POLICY_LRFU) {
            float v = pol[e] * w;
            if (selected[e]) v = v + 1.0f;
            pol[e] = v;
        }
    }
}

/* zR, zT, zS: [S][L][N] fp32 logits of this token (zR already includes any
 * bias; zT is read only with the router policy in the Temporal and
 * Spatio-Temporal modes, zS only in the modes with a Spatio Router).
 * Returns 0, or -1 on a broken invariant. */
int orc_step(const orc_cfg* c, orc_state* st, const float* zR, const float* zT, const float* zS,
             orc_out* out) {
    const int L = c->L, N = c->N, K = c->K, S = c->S;
    const int spatio = c->mode == ORC_MODE_SPATIO_TEMPORAL || c->mode == ORC_MODE_SPATIO_ONLY;
    const int router_policy = c->policy == ORC_POLICY_ROUTER;
    const int t = st->t;
    const int counted = t >= c->warmup_tokens;
    float pR[ORC_NMAX], pT[ORC_NMAX], pSn[ORC_NMAX], sT[ORC_NMAX], sST[ORC_NMAX];
    int32_t sel[ORC_NMAX];
    for (int l = 0; l < L; ++l) {
        /* Pre-access refinement (Algorithm 2): needs the previous token's
         * same-layer scores, so it starts at t = 1. */
        if (spatio && t >= 1 && c->R > 0) {
            for (int s = 0; s < S; ++s) {
                const size_t sl = (size_t)s * L + l;
                /* p^R_{t-1,l} + p^T_{t-1,l} (Spatio-Temporal) or p^R_{t-1,l}
                 * (Spatio-only) */
                const float* aT = st->aT + sl * N;
                const float* pred = st->pS + (size_t)s * N; /* p^S at rho(t,l) */
                for (int e = 0; e < N; ++e) sST[e] = aT[e] + pred[e];
                int32_t loaded[ORC_NMAX];
                int nP = orc_refine(st->cache + sl * N, N, c->C, sST, c->R, loaded);
                if (c->policy == ORC_POLICY_LRU)   /* inserted as the most recently used */
                    for (int i = 0; i < nP; ++i) st->pol[sl * N + loaded[i]] = (float)(2 * t + 1);
                if (counted) st->ctr[sl * ORC_NCTR + ORC_CTR_P] += nP;
                if (out && out->nP) out->nP[sl] = nP;
                if (out && out->sST) memcpy(out->sST + sl * N, sST, sizeof(float) * (size_t)N);
            }
            int f = orc_residency(c, st, l, NULL);
            if (f < 0) return -1;
            if (counted) st->phys[(size_t)l * 2 + 1] += f;
            if (out && out->fills) out->fills[l * 2 + 1] = f;
        } else {
            for (int s = 0; s < S; ++s) {
                if (out && out->nP) out->nP[(size_t)s * L + l] = 0;
            }
            if (out && out->fills) out->fills[l * 2 + 1] = 0;
        }
        /* Native routing, access, post-access retention (Algorithm 1). */
        uint8_t executed[ORC_NMAX];   /* experts this layer step's FFN executes */
        memset(executed, 0, (size_t)N);
        for (int s = 0; s < S; ++s) {
            const size_t sl = (size_t)s * L + l;
            orc_softmax(zR + sl * N, N, pR);
            orc_topk(zR + sl * N, N, K, sel);
            for (int k = 0; k < K; ++k) executed[sel[k]] = 1;
            double gsum = 0.0;
            for (int k = 0; k < K; ++k) gsum += (double)pR[sel[k]];
            if (router_policy) {
                orc_softmax(zT + sl * N, N, pT);
                for (int e = 0; e < N; ++e) sT[e] = pR[e] + pT[e];
            } else {
                uint8_t selected[ORC_NMAX];
                memset(selected, 0, (size_t)N);
                for (int k = 0; k < K; ++k) selected[sel[k]] = 1;
                orc_policy_access(c->policy, c->lrfu_w, st->pol + sl * N, N, selected, t);
                memcpy(sT, st->pol + sl * N, sizeof(float) * (size_t)N);
            }
            uint8_t* cache = st->cache + sl * N;
            int hits = 0;
            for (int k = 0; k < K; ++k) hits += cache[sel[k]] ? 1 : 0;
            int nD = orc_update_cache(cache, N, c->C, sel, K, sT, NULL);
            if (hits + nD != K) return -1;
            if (orc_count(cache, N) > c->C) return -1;
            if (spatio) {
                /* the next token's a-score for this layer */
                memcpy(st->aT + sl * N, c->mode == ORC_MODE_SPATIO_ONLY ? pR : sT, sizeof(float) * (size_t)N);
                orc_softmax(zS + sl * N, N, pSn);
                memcpy(st->pS + (size_t)s * N, pSn, sizeof(float) * (size_t)N);
            }
            if (counted) {
                for (int k = 0; k < K; ++k) st->selcount[(size_t)l * N + sel[k]] += 1;
                int64_t* ctr = st->ctr + sl * ORC_NCTR;
                ctr[ORC_CTR_A] += K;
                ctr[ORC_CTR_HITS] += hits;
                ctr[ORC_CTR_D] += nD;
                ctr[ORC_CTR_T] += 1;
            }
            if (out) {
                if (out->sel) memcpy(out->sel + sl * K, sel, sizeof(int32_t) * (size_t)K);
                if (out->gate)
                    for (int k = 0; k < K; ++k) out->gate[sl * K + k] = (double)pR[sel[k]] / gsum;
                if (out->pR) memcpy(out->pR + sl * N, pR, sizeof(float) * (size_t)N);
                if (out->sT) memcpy(out->sT + sl * N, sT, sizeof(float) * (size_t)N);
                if (out->hits) out->hits[sl] = hits;
                if (out->nD) out->nD[sl] = nD;
            }
        }
        int f = orc_residency(c, st, l, executed);
        if (f < 0) return -1;
        if (counted) st->phys[(size_t)l * 2 + 0] += f;
        if (out && out->fills) out->fills[l * 2 + 0] = f;
    }
    st->t = t + 1;
    return 0;
}
