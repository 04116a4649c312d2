// fill.hip - physical residency and expert copies (the demand loads and
// proactive loads of Section 2 / Algorithm 2 as transfers into HBM slots).
//
// One launch handles one residency event of one layer: after the post-access
// update (demand loads) or after refinement (proactive loads), the layer's
// HBM slots must hold the union U of the streams' caches.  Experts that left
// U free their slot; each new expert, in ascending order, takes the lowest
// free slot and is copied there from the cold pool.
//
// Every workgroup derives the same assignment from the same inputs (the
// caches and the slot maps of version rv, which nobody writes during the
// launch), then copies its share of the new experts; workgroup 0 also writes
// the new slot maps (version rv ^ 1) and, after the post-access update, lays
// out the layer step's FFN work units.  No workgroup waits for another, and
// the host never has to read the fill list.  The pool may be pinned host
// memory mapped into the device; copies then run over the host link.
#include "cmoe_internal.h"

namespace cmoe {

namespace {

// Threads of a fill workgroup (four wavefronts), a compile-time constant so
// that no loop bound has to be read from the dispatch packet.
constexpr int kFillThreads = 256;

// Block-wide exclusive prefix counts and sums over the 256 threads of the
// block, each call with one barrier: the wavefront totals go to LDS slots
// (four per value), and consecutive calls use different slots, so no barrier
// is needed after one call before the next.
// NF flags at once: the ballot bits below the lane; total[f] gets the block
// total of flag f.  slot: 4 NF ints.
template <int NF>
__device__ void block_counts(const bool (&v)[NF], int (&below)[NF], int (&total)[NF], int* slot) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
    for (int f = 0; f < NF; ++f) {
        const unsigned long long b = __ballot(v[f]);
        below[f] = (int)__builtin_amdgcn_mbcnt_hi((unsigned)(b >> 32), __builtin_amdgcn_mbcnt_lo((unsigned)b, 0u));
        if (lane == 0) slot[4 * f + w] = __popcll(b);
    }
    __syncthreads();
#pragma unroll
    for (int f = 0; f < NF; ++f) {
        int off = 0, tot = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            if (i < w) off += slot[4 * f + i];
            tot += slot[4 * f + i];
        }
        below[f] += off;
        total[f] = tot;
    }
}

// Values: an inclusive wavefront scan in DPP steps (shifts by 1, 2, 4 and 8
// inside each 16-lane row, then the last lane of row 0 and of row 1 added to
// the rows after them); a lane whose source is outside its row adds 0.
__device__ int block_scan(int v, int* total, int* slot) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    int x = v;
    x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xF, 0xF, false);  // row_shr:1
    x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xF, 0xF, false);  // row_shr:2
    x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xF, 0xF, false);  // row_shr:4
    x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xF, 0xF, false);  // row_shr:8
    x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xA, 0xF, false);  // row_bcast:15 into rows 1, 3
    x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xC, 0xF, false);  // row_bcast:31 into rows 2, 3
    if (lane == 63) slot[w] = x;
    __syncthreads();
    int off = 0, tot = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        if (i < w) off += slot[i];
        tot += slot[i];
    }
    *total = tot;
    return off + x - v;
}

// bf16 experts are stored in their HBM slot in the order the FFN kernels
// consume them, so that every load instruction reads 1 KB of contiguous
// memory.  Units are 16 bytes (8 bf16); lane l of a wavefront takes unit l of
// a 64-unit run.
//   gate/up part, units [0, F d / 4):
//     ((((ft * (d/64) + c) * 2 + mat) * 2 + half) * 64 + lane)
//     = W_mat[16 ft + lane % 16][64 c + 32 half + 8 (lane / 16) .. + 8],
//     mat 0 = gate, 1 = up
//   down part, units [F d / 4, 3 F d / 8):
//     F d / 4 + ((((dt * (F/64) + c) * 2 + mt) * 2 + half) * 64 + lane)
//     = W_down[32 dt + 16 mt + lane % 16][64 c + 32 half + 8 (lane / 16) .. + 8]
// The cold pool keeps the plain row-major layout.  Every 128-unit block of
// the packed order (one run for each half) holds 16 source rows x 128
// contiguous bytes: rows 16 ft + r of W_mat at columns 64 c .. 64 c + 63 for
// the gate/up part, rows 32 dt + 16 mt + r of W_down at columns 64 c .. for
// the down part.  Two copy orders give the same result:
//   - block order (pool in HBM): walk the packed blocks, 8 consecutive lanes
//     reading one 128-byte row segment, and write each block's contiguous
//     2 KB;
//   - source order (pool in pinned host memory): walk the source in its own
//     order, so each wavefront reads 1 KB of one row.  Reads over the host
//     link are then long requests (56 GB/s measured on MI355X, against 42 GB/s
//     for 128-byte segments).  Each 16-byte unit is scattered to its packed
//     position; the L2 merges the partial lines.
struct BlockMap {
    int64_t src;  // source unit of row 0, chunk 0 of the block
    int64_t row;  // source units between consecutive rows
};

__device__ inline BlockMap packed_block(int b, int d, int F) {
    const int partA = F / 16 * (d / 64) * 2;  // gate/up blocks
    BlockMap m;
    if (b < partA) {
        const int sub = b & 1;  // gate or up
        const int t = b >> 1;
        const int c = t % (d / 64), tile = t / (d / 64);
        m.src = ((int64_t)sub * F * d + (int64_t)16 * tile * d + 64 * c) / 8;
        m.row = d / 8;
    } else {
        const int v = b - partA;
        const int sub = v & 1;  // 16-row half of the 32-row tile
        const int t = v >> 1;
        const int c = t % (F / 64), tile = t / (F / 64);
        m.src = (2 * (int64_t)F * d + (int64_t)(32 * tile + 16 * sub) * F + 64 * c) / 8;
        m.row = F / 8;
    }
    return m;
}

// Source unit w of a block (row w / 8, 16-byte chunk w % 8 of the row's 128
// bytes) goes to packed unit (chunk / 4) * 64 + row + 16 (chunk % 4).
__device__ inline int packed_dest_in_block(int w) {
    const int r = w >> 3, j = w & 7;
    return (j >> 2) * 64 + r + 16 * (j & 3);
}

// Packed position of source unit i of an expert (row-major W_gate, W_up,
// then W_down, 16-byte units): the inverse of the block order above.
__device__ inline int64_t packed_of_source(int64_t i, int d, int F) {
    const int ud = d / 8, uf = F / 8;      // units per row
    const int64_t nA = (int64_t)F * ud;    // units of W_gate (and of W_up)
    if (i < 2 * nA) {
        const int mat = i >= nA;
        const int64_t k = i - mat * nA;
        const int row = (int)(k / ud), u = (int)(k - (int64_t)row * ud);
        const int64_t b = ((int64_t)(row >> 4) * (ud / 8) + (u >> 3)) * 2 + mat;
        return b * 128 + packed_dest_in_block(((row & 15) << 3) | (u & 7));
    }
    const int64_t k = i - 2 * nA;
    const int row = (int)(k / uf), u = (int)(k - (int64_t)row * uf);
    const int64_t b = ((int64_t)(row >> 5) * (uf / 8) + (u >> 3)) * 2 + ((row >> 4) & 1);
    return 2 * nA + b * 128 + packed_dest_in_block(((row & 15) << 3) | (u & 7));
}

// Cache word i = s NW + j: word j of stream s's membership bits of the layer.
__device__ inline unsigned long long cache_word(const Layout& lo, int layer, int i) {
    const int s = i / lo.NW, j = i - s * lo.NW;
    return lo.cache[((int64_t)s * lo.L + layer) * lo.NW + j];
}

// Workgroup-local state of one residency event.
struct FillLds {
    unsigned long long U[4];
    int so[kMaxN], se[kMaxN], stp[kMaxN], rnd_s[kMaxN], free_list[kMaxN], enter_list[kMaxN], victim_list[kMaxN];
    int lds4[4];       // block-scan slots
    int lds_cnt[2][12];  // block-count slots: round plan; free slots, entries, multi-pass units
    __align__(16) int key[kMaxN];
    int by_rank[kMaxN], who[kMaxN], m_rank[kMaxN];
};

// One residency event (or one FFN round of one), run by nwg workgroups of the
// launch, this one being number wg; returns once its share of the copies is
// done.  Workgroup 0 of the event writes the new slot maps and work units.
__device__ __forceinline__ void residency_event(const Layout& lo, const FillArgs& f, FillLds& sm, int wg, int nwg) {
    unsigned long long* U = sm.U;
    int *so = sm.so, *se = sm.se, *stp = sm.stp, *rnd_s = sm.rnd_s, *free_list = sm.free_list;
    int *enter_list = sm.enter_list, *victim_list = sm.victim_list, *lds4 = sm.lds4;
    const int tid = threadIdx.x;
    const int N = lo.N, layer = f.layer, P = lo.n_slots;
    const int64_t vin = (int64_t)f.rv * lo.L + layer, vout = (int64_t)(f.rv ^ 1) * lo.L + layer;
    const int32_t* so_in = lo.slot_of + vin * N;
    const int32_t* se_in = lo.slot_exp + vin * P;
    const int32_t* st_in = lo.slot_stamp + vin * P;
    const bool demand = f.kind == 0;
    // Every global load of the prologue is issued before the first is used,
    // whatever the event (indices clamped; a value that is not needed is not
    // used): the slot maps and stamps, the bucket sizes (the executed experts
    // and the FFN work units), the round plan of a later round, the fill
    // counters workgroup 0 adds to, and the first batch of cache words.
    const bool units = demand && f.units && wg == 0;
    const int S_NW = lo.S * lo.NW;
    const int so_v = so_in[min(tid, N - 1)];
    const int se_v = se_in[min(tid, P - 1)];
    const int st_v = st_in[min(tid, P - 1)];
    const int mb_v = lo.bcount[(int64_t)f.bbuf * N + min(tid, N - 1)];
    const int ro_v = lo.round_of[min(tid, N - 1)];
    const int64_t phys_v = lo.phys[layer * 2 + f.kind];
    const int32_t sf_v = lo.step_fills[layer * 2];
    constexpr int kWords = 4;  // cache words per thread per batch
    unsigned long long w[kWords];
#pragma unroll
    for (int u = 0; u < kWords; ++u) w[u] = cache_word(lo, layer, min(tid + u * kFillThreads, S_NW - 1));
    __builtin_amdgcn_sched_barrier(0);
    if (tid < 4) U[tid] = 0ull;
    if (tid < N) so[tid] = so_v;
    if (tid < P) {
        se[tid] = se_v;
        stp[tid] = st_v;
    }
    __syncthreads();
    for (int i0 = 0; i0 < S_NW; i0 += kWords * kFillThreads) {
        if (i0 > 0) {
#pragma unroll
            for (int u = 0; u < kWords; ++u)
                w[u] = cache_word(lo, layer, min(i0 + tid + u * kFillThreads, S_NW - 1));
            __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int u = 0; u < kWords; ++u) {
            const int i = i0 + tid + u * kFillThreads;
            if (i < S_NW && w[u]) atomicOr(&U[i % lo.NW], w[u]);
        }
    }
    __syncthreads();
    const int m_v = demand ? mb_v : 0;
    const int e = tid;
    const bool inU = e < N && ((U[e >> 6] >> (e & 63)) & 1ull);
    int cur = e < N ? so[e] : -1;
    if (e < N && cur >= 0 && !inU) {  // left every cache: free its slot
        se[cur] = -1;
        so[e] = -1;
        cur = -1;
    }
    int nU = 0;
    for (int j = 0; j < lo.NW; ++j) nU += __popcll(U[j]);
    const bool overflow = nU > P;  // the union does not fit the arena (block-uniform)
    __syncthreads();
    // FFN round of each expert the layer step executes.  While the union fits,
    // all run in round 0.  Otherwise round 0 plans the rounds: the executed
    // experts already resident first, then the others, each group ascending,
    // P per round; later rounds read the plan.
    const bool inE = demand && e < N && m_v > 0;
    int rnd = -1;
    if (demand) {
        if (!overflow) {
            rnd = inE ? 0 : -1;
        } else if (f.round == 0) {
            const bool res_e = inE && cur >= 0, mis_e = inE && cur < 0;
            const bool fl[2] = {res_e, mis_e};
            int rk[2], n[2];
            block_counts<2>(fl, rk, n, sm.lds_cnt[0]);
            rnd = res_e ? rk[0] / P : (mis_e ? (n[0] + rk[1]) / P : -1);
        } else {
            rnd = e < N ? ro_v : -1;
        }
    }
    if (e < N) rnd_s[e] = rnd;
    const bool now = demand && rnd >= 0 && rnd == f.round;  // executed in this round
    bool enter;
    if (!demand) enter = e < N && inU && cur < 0;
    else if (!overflow) enter = f.round == 0 && e < N && inU && cur < 0;
    else enter = now && cur < 0;
    const bool is_free = tid < P && se[tid] == -1;
    // The work units of this round (below) need to know whether any bucket
    // takes more than one pass, and rank the experts by their bucket sizes
    // if one does: the flag joins the free-slot and entry counts, and the
    // ranking keys are stored before the same barrier.
    const int m_own = (units && now) ? m_v : 0;
    const int ut = lo.unit_tokens;
    const int mykey = (m_own << 8) | (255 - tid);
    if (units) sm.key[tid] = tid < N ? mykey : -1;  // kFillThreads == kMaxN: every entry is written
    const bool fl[3] = {is_free, enter, units && m_own > ut};
    int rk[3], n[3];
    block_counts<3>(fl, rk, n, sm.lds_cnt[1]);
    const int rf = rk[0], re = rk[1], nfree = n[0], nenter = n[1];
    const bool multi = n[2] > 0;
    if (is_free) free_list[rf] = tid;
    // A round that needs more than the free slots evicts the least recently
    // used experts that no remaining round needs (lower slot on ties), ranked
    // by (stamp, slot); after refinement only free slots are filled.
    int nvict = 0;
    if (demand && overflow && nenter > nfree) {  // block-uniform
        bool vict = false;
        int rank = 0;
        if (tid < P && se[tid] >= 0) {
            vict = rnd_s[se[tid]] < f.round;
            if (vict) {
                const int sq = stp[tid];
                for (int q2 = 0; q2 < P; ++q2) {
                    const int v2 = se[q2];
                    if (v2 < 0 || rnd_s[v2] >= f.round) continue;
                    const int s2 = stp[q2];
                    rank += (s2 < sq || (s2 == sq && q2 < tid)) ? 1 : 0;
                }
            }
        }
        if (vict) victim_list[rank] = tid;
        nvict = __syncthreads_count(vict);
    }
    const int nent = (!demand && overflow) ? min(nenter, nfree) : nenter;
    __syncthreads();
    const bool takes = enter && re < nent;
    if (takes) {  // rank re among new experts takes the rank-re free slot, then the victims in rank order
        int q = -1;
        if (re < nfree)
            q = free_list[re];
        else if (re - nfree < nvict)
            q = victim_list[re - nfree];
        if (q >= 0) {
            if (re >= nfree) so[se[q]] = -1;  // evicted
            so[e] = q;
            se[q] = e;
        }
        enter_list[re] = q >= 0 ? e : -1;  // q < 0 cannot happen: a round fits the arena
    }
    __syncthreads();
    // last use: the experts executed in this round and every expert copied in
    if (e < N && (now || takes) && so[e] >= 0) stp[so[e]] = f.clk;
    __syncthreads();
    if (wg == 0) {
        int32_t* so_out = lo.slot_of + vout * N;
        int32_t* se_out = lo.slot_exp + vout * P;
        int32_t* st_out = lo.slot_stamp + vout * P;
        if (tid < N) so_out[tid] = so[tid];
        if (tid < P) {
            se_out[tid] = se[tid];
            st_out[tid] = stp[tid];
        }
        if (demand && f.round == 0 && tid < N) lo.round_of[tid] = rnd;
        if (tid == 0) {
            if (demand && f.round > 0)
                lo.step_fills[layer * 2] = sf_v + nent;
            else
                lo.step_fills[layer * 2 + f.kind] = nent;
            if (f.zero_pre) lo.step_fills[layer * 2 + 1] = 0;
            if (f.counted) lo.phys[layer * 2 + f.kind] = phys_v + nent;
        }
    }
    // FFN work units of this round: each of its experts' buckets cut into
    // passes of up to lo.unit_tokens tokens, each stored with its expert's new
    // slot and its token count, so that an FFN wavefront finds all three with
    // one load.  When no bucket needs a second pass, unit e is expert e (or
    // none if it has no tokens in this round).
    int4* unit4 = reinterpret_cast<int4*>(lo.units);
    if (units && !multi) {
        // kFillThreads >= N: thread e holds expert e's bucket size
        for (int i = tid; i < lo.max_units; i += kFillThreads)
            unit4[i] = (i < N && m_own > 0) ? int4{i, so[i], m_own, 0} : int4{-1, -1, 0, 0};
    } else if (units) {
        // otherwise experts with more tokens go first (lower index on ties),
        // so the longest units start first.  Rank of expert e = number of
        // larger keys (m << 8) | (255 - e), all distinct.
        // (the keys were stored before the barrier of the counts above)
        int *by_rank = sm.by_rank, *who = sm.who, *m_rank = sm.m_rank;
        const int m = m_own;
        int rank = 0;
        if (tid < N) {
            // batches of 32 keys, every LDS read of a batch issued before the
            // first compare; keys past N are -1 and never counted
            const int4* k4 = reinterpret_cast<const int4*>(sm.key);
            for (int u0 = 0; u0 < (N + 3) / 4; u0 += 8) {  // u0 + 7 < kMaxN / 4
                int4 v[8];
#pragma unroll
                for (int i = 0; i < 8; ++i) v[i] = k4[u0 + i];
#pragma unroll
                for (int i = 0; i < 8; ++i)
                    rank += (v[i].x > mykey) + (v[i].y > mykey) + (v[i].z > mykey) + (v[i].w > mykey);
            }
        }
        if (tid < N) {
            by_rank[rank] = (m + ut - 1) / ut;
            who[rank] = tid;
            m_rank[rank] = m;
        }
        __syncthreads();
        const int passes = tid < N ? by_rank[tid] : 0;
        int total;
        const int off = block_scan(passes, &total, lds4);
        if (tid < N) {
            const int e = who[tid];
            for (int q = 0; q < passes; ++q)
                unit4[off + q] = int4{(q << 8) | e, so[e], min(ut, m_rank[tid] - ut * q), 0};
        }
        for (int i = total + tid; i < lo.max_units; i += kFillThreads) unit4[i] = int4{-1, -1, 0, 0};
    }
    if (nent == 0) return;
    const int64_t bytes = lo.expert_elems * (lo.dtype == 1 ? 2 : 4);
    const int64_t n16 = bytes / 16;
    const int64_t gid = (int64_t)wg * kFillThreads + tid;
    const int64_t gs = (int64_t)nwg * kFillThreads;
    for (int k = 0; k < nent; ++k) {
        const int ex = enter_list[k];
        if (ex < 0) continue;
        const int q = so[ex];
        const uint4* src =
            reinterpret_cast<const uint4*>(static_cast<const char*>(lo.pool) + ((int64_t)layer * N + ex) * bytes);
        uint4* dst = reinterpret_cast<uint4*>(static_cast<char*>(lo.arena) + ((int64_t)layer * lo.n_slots + q) * bytes);
        if (lo.dtype == 1 && lo.pool_host) {
            for (int64_t i = gid; i < n16; i += gs) dst[packed_of_source(i, lo.d, lo.F)] = src[i];
        } else if (lo.dtype == 1) {
            for (int64_t i = gid; i < n16; i += gs) {
                const int b = (int)(i >> 7), w = (int)(i & 127);
                const BlockMap m = packed_block(b, lo.d, lo.F);
                dst[(int64_t)b * 128 + packed_dest_in_block(w)] = src[m.src + (w >> 3) * m.row + (w & 7)];
            }
        } else {
            // fp32: each matrix transposed (W_gate^T, W_up^T [d][F], W_down^T
            // [F][d]) so that the lanes of the FFN kernels, one output row
            // each, read consecutive addresses; walked in source order
            const float* s32 = reinterpret_cast<const float*>(src);
            float* d32 = reinterpret_cast<float*>(dst);
            const int64_t dF = (int64_t)lo.d * lo.F;
            for (int64_t i = gid; i < 3 * dF; i += gs) {
                const int part = (int)(i / dF);
                const int64_t r = i - part * dF;
                int64_t o;
                if (part < 2) {
                    const int64_t f = r / lo.d, k = r - f * lo.d;  // W[f][k]
                    o = part * dF + k * lo.F + f;
                } else {
                    const int64_t j = r / lo.F, f = r - j * lo.F;  // W_down[j][f]
                    o = 2 * dF + f * lo.d + j;
                }
                d32[o] = s32[i];
            }
        }
    }
}

// One residency event, or two of different layers (g.layer >= 0): the
// demand event of one layer and the proactive event of the next, which both
// follow the same cache step, in one launch, each on half the workgroups
// (even ones: f, odd ones: g).
__global__ __launch_bounds__(kFillThreads) void fill_kernel(Layout lo, FillArgs f, FillArgs g) {
    __shared__ FillLds sm;
    if (g.layer < 0)
        residency_event(lo, f, sm, blockIdx.x, gridDim.x);
    else if ((blockIdx.x & 1) == 0)
        residency_event(lo, f, sm, blockIdx.x >> 1, (gridDim.x + 1) >> 1);
    else
        residency_event(lo, g, sm, blockIdx.x >> 1, gridDim.x >> 1);
}

}  // namespace

hipError_t launch_fill(const Layout& lo, const FillArgs& f, const FillArgs* g, hipStream_t st, const Timing& tm) {
    FillArgs none{};
    none.layer = -1;
    launch_kernel(fill_kernel, dim3(lo.pool_host ? kFillBlocksHost : kFillBlocksDevice), dim3(kFillThreads), st, tm, lo, f,
                  g ? *g : none);
    return hipGetLastError();
}

}  // namespace cmoe
