// router.hip - router logits z = W h for the native, Temporal and Spatio
// routers of one layer (Section 2: W^R h; Section 3.2: W^T h; Section 3.3:
// W^S h), all streams at once.
//
// The logits decide expert selection and cache priorities, so they are
// summed in fp64 and rounded to fp32 once (after the bias), like the plain
// definition: the fp32 result then differs from an fp64 sequential sum only
// when that sum lies within ~1e-16 relative of an fp32 rounding boundary.
//
// Work split: one workgroup per 16 experts x 16 streams x one d-range
// (split-K, at most kMaxSplit splits), on the fp64 matrix core
// (v_mfma_f64_16x16x4_f64).  The range is cut into kRouterWaves consecutive
// sub-ranges, one per wavefront; the wavefronts' tiles are added in LDS in
// wavefront order and the workgroup writes one partial.  The cache-step
// kernel adds the partials of each logit in ascending split order, adds the
// native bias and rounds once, so the result does not depend on the order in
// which workgroups finish.  Each lane loads 8 consecutive weights (and hidden
// values) at once; the four lane groups of an MFMA take k-slots base + 8 g + j
// for step j, the same permutation for both operands, so every product pairs
// W[e][i] with h[s][i].
#include "cmoe_internal.h"

namespace cmoe {

typedef double f64x4 __attribute__((ext_vector_type(4)));

// 8 consecutive values of a row as loaded (one 16-byte load for bf16, two
// for fp32), then widened exactly to fp64.
template <bool BF16>
struct Raw8 {
    uint4 v[BF16 ? 1 : 2];
};

template <bool BF16>
__device__ inline Raw8<BF16> load8(const void* base, int64_t idx) {
    Raw8<BF16> r;
    if constexpr (BF16) {
        r.v[0] = *reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(base) + idx);
    } else {
        const uint4* p = reinterpret_cast<const uint4*>(reinterpret_cast<const float*>(base) + idx);
        r.v[0] = p[0];
        r.v[1] = p[1];
    }
    return r;
}

template <bool BF16>
__device__ inline void widen8(const Raw8<BF16>& r, double* out) {
    uint32_t w[8];
    if constexpr (BF16) {
        const uint32_t p[4] = {r.v[0].x, r.v[0].y, r.v[0].z, r.v[0].w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            w[2 * j] = p[j] << 16;
            w[2 * j + 1] = p[j] & 0xFFFF0000u;
        }
    } else {
        const uint32_t p[8] = {r.v[0].x, r.v[0].y, r.v[0].z, r.v[0].w, r.v[1].x, r.v[1].y, r.v[1].z, r.v[1].w};
#pragma unroll
        for (int j = 0; j < 8; ++j) w[j] = p[j];
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) out[j] = (double)__uint_as_float(w[j]);
}

// Loads of chunks c0 .. c0 + KB - 1, clamped to the wavefront's last chunk
// (the re-read of a clamped chunk is never used).
template <bool BF16, int KB>
__device__ inline void issue_batch(const void* W, const void* h, int64_t arow, int64_t brow, int c0, int nch,
                                   Raw8<BF16>* ra, Raw8<BF16>* rb) {
#pragma unroll
    for (int u = 0; u < KB; ++u) {
        const int c = min(c0 + u, nch - 1);
        ra[u] = load8<BF16>(W, arow + c * 32);
        rb[u] = load8<BF16>(h, brow + c * 32);
    }
}

// Widening and matrix-core work of the chunks of a batch that lie in range,
// in ascending k order (a wavefront-uniform test).
template <bool BF16, int KB>
__device__ inline void mfma_batch(const Raw8<BF16>* ra, const Raw8<BF16>* rb, int c0, int nch, f64x4& acc) {
#pragma unroll
    for (int u = 0; u < KB; ++u) {
        if (c0 + u < nch) {
            double av[8], bv[8];
            widen8<BF16>(ra[u], av);
            widen8<BF16>(rb[u], bv);
#pragma unroll
            for (int j = 0; j < 8; ++j) acc = __builtin_amdgcn_mfma_f64_16x16x4f64(av[j], bv[j], acc, 0, 0, 0);
        }
    }
}

// grid: x = n_r * ceil(N/16) * ceil(S/16), z = nsplit; block: kRouterWaves
// wavefronts; KB = k chunks whose loads are issued together (at most the
// chunks of a wavefront's range)
template <bool BF16, int KB>
__global__ __launch_bounds__(64 * kRouterWaves) void router_kernel(Layout lo, int l, const void* h, int dk) {
    __shared__ f64x4 red[kRouterWaves - 1][64];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int r16 = lane & 15, g = lane >> 4;
    const int et_n = (lo.N + 15) / 16, st_n = (lo.S + 15) / 16;
    int b = blockIdx.x;
    const int st = b % st_n;
    b /= st_n;
    const int et = b % et_n;
    const int r = b / et_n;
    const int p = blockIdx.z;
    const int i0 = (p * kRouterWaves + wv) * dk;
    const int nch = i0 < lo.d ? (min(i0 + dk, lo.d) - i0) / 32 : 0;  // 32-wide k chunks of this wavefront

    const int e_a = et * 16 + r16;  // expert row this lane feeds into A
    const int s_b = st * 16 + r16;  // stream column this lane feeds into B
    const bool va = e_a < lo.N, vb = s_b < lo.S;
    const void* W = lo.rw[r];
    const int64_t arow = ((int64_t)l * lo.N + (va ? e_a : 0)) * lo.d + i0 + 8 * g;
    const int64_t brow = ((int64_t)(vb ? s_b : 0) * lo.L + l) * lo.d + i0 + 8 * g;

    // Every load of a batch is issued before the first is used.  Rows past N
    // or S read row 0: they only feed output rows and columns that are never
    // stored.
    const int nchu = __builtin_amdgcn_readfirstlane(nch);
    f64x4 acc = {0.0, 0.0, 0.0, 0.0};
    for (int c0 = 0; c0 < nchu; c0 += KB) {
        Raw8<BF16> ra[KB], rb[KB];
        issue_batch<BF16, KB>(W, h, arow, brow, c0, nchu, ra, rb);
        __builtin_amdgcn_sched_barrier(0);
        mfma_batch<BF16, KB>(ra, rb, c0, nchu, acc);
    }
    // the workgroup's sub-range tiles, added in wavefront order
    if (wv > 0) red[wv - 1][lane] = acc;
    __syncthreads();
    if (wv > 0) return;
#pragma unroll
    for (int w = 0; w < kRouterWaves - 1; ++w) {
        const f64x4 o = red[w][lane];
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[q] = acc[q] + o[q];
    }
    // Output of the fp64 16x16x4 MFMA: lane (r16, g) holds D[g + 4 q][r16] in
    // acc[q], i.e. expert row g + 4 q of the tile, stream column r16.  The
    // partial of split p goes to zpart[s][r][e][p] (p padded to zstride): the
    // splits of one logit are contiguous for the cache-step kernel, which adds
    // them in order.
    const int s = st * 16 + r16;
    if (s < lo.S) {
        double* out = lo.zpart + ((int64_t)s * lo.n_r + r) * lo.N * lo.zstride + p;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = et * 16 + g + 4 * q;
            if (e < lo.N) out[(int64_t)e * lo.zstride] = acc[q];
        }
    }
}

template <bool BF16>
static void launch_router_t(const Layout& lo, int l, const void* h, hipStream_t st, const Timing& tm) {
    const int dk = lo.rdk;  // multiple of 32; the last split may be shorter (d % 32 == 0)
    const dim3 grid(lo.n_r * ((lo.N + 15) / 16) * ((lo.S + 15) / 16), 1, lo.nsplit);
    const dim3 block(64 * kRouterWaves);
    const int cpw = dk / 32;  // k chunks per wavefront
    if (cpw >= 4)
        launch_kernel(router_kernel<BF16, 4>, grid, block, st, tm, lo, l, h, dk);
    else if (cpw >= 2)
        launch_kernel(router_kernel<BF16, 2>, grid, block, st, tm, lo, l, h, dk);
    else
        launch_kernel(router_kernel<BF16, 1>, grid, block, st, tm, lo, l, h, dk);
}

hipError_t launch_router(const Layout& lo, int l, const void* h, hipStream_t st, const Timing& tm) {
    if (lo.dtype == 1)
        launch_router_t<true>(lo, l, h, st, tm);
    else
        launch_router_t<false>(lo, l, h, st, tm);
    return hipGetLastError();
}

}  // namespace cmoe
