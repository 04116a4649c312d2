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

__device__ inline void load8_as_f64(const void* base, int64_t idx, bool bf16, bool valid, double* out) {
    // 8 consecutive values widened exactly to fp64
    if (!valid) {
#pragma unroll
        for (int j = 0; j < 8; ++j) out[j] = 0.0;
        return;
    }
    if (bf16) {
        const uint4 v = *reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(base) + idx);
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            out[2 * j] = (double)__uint_as_float(w[j] << 16);
            out[2 * j + 1] = (double)__uint_as_float(w[j] & 0xFFFF0000u);
        }
    } else {
        const float4* p = reinterpret_cast<const float4*>(reinterpret_cast<const float*>(base) + idx);
        const float4 a = p[0], b = p[1];
        out[0] = a.x; out[1] = a.y; out[2] = a.z; out[3] = a.w;
        out[4] = b.x; out[5] = b.y; out[6] = b.z; out[7] = b.w;
    }
}

// grid: x = n_r * ceil(N/16) * ceil(S/16), z = nsplit; block: kRouterWaves wavefronts
template <bool BF16>
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

    f64x4 acc = {0.0, 0.0, 0.0, 0.0};
    constexpr int kBatch = 4;  // chunks whose loads are issued together
    for (int c0 = 0; c0 < nch; c0 += kBatch) {
        double av[kBatch][8], bv[kBatch][8];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const bool in = c0 + u < nch;
            load8_as_f64(W, arow + (c0 + u) * 32, BF16, va && in, av[u]);
            load8_as_f64(h, brow + (c0 + u) * 32, BF16, vb && in, bv[u]);
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u)
#pragma unroll
            for (int j = 0; j < 8; ++j) acc = __builtin_amdgcn_mfma_f64_16x16x4f64(av[u][j], bv[u][j], acc, 0, 0, 0);
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

hipError_t launch_router(const Layout& lo, int l, const void* h, hipStream_t st) {
    const int dk = lo.rdk;  // multiple of 32; the last split may be shorter (d % 32 == 0)
    const int tiles = lo.n_r * ((lo.N + 15) / 16) * ((lo.S + 15) / 16);
    if (lo.dtype == 1)
        hipLaunchKernelGGL(router_kernel<true>, dim3(tiles, 1, lo.nsplit), dim3(64 * kRouterWaves), 0, st, lo, l, h,
                           dk);
    else
        hipLaunchKernelGGL(router_kernel<false>, dim3(tiles, 1, lo.nsplit), dim3(64 * kRouterWaves), 0, st, lo, l, h,
                           dk);
    return hipGetLastError();
}

}  // namespace cmoe
