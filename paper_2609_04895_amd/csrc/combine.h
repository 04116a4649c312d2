// combine.h - the gated combine of one layer's expert outputs, as a device
// function: y[s][l] = sum over k of the gated outputs yp[s][k] (the gates
// are already applied by the down projection), added in k order in fp32.
// Used by the stand-alone combine kernel and by the cache-step launch of the
// next layer, which runs it in workgroups of its own.
#pragma once

#include <type_traits>

#include "cmoe_internal.h"

namespace cmoe {

constexpr int kCombineThreads = 256;  // threads per combine workgroup

// Four consecutive gated outputs in fp32: bf16 ones widened exactly.
template <bool BF16>
struct Quad {
    using Raw = typename std::conditional<BF16, uint2, float4>::type;
    __device__ static float4 widen(const Raw& v) {
        if constexpr (BF16)
            return make_float4(__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xFFFF0000u),
                               __uint_as_float(v.y << 16), __uint_as_float(v.y & 0xFFFF0000u));
        else
            return v;
    }
};

template <bool BF16>
__device__ inline void combine_quad_t(const Layout& lo, int l, float* __restrict__ y, int s, int c) {
    using Raw = typename Quad<BF16>::Raw;
    const int n4 = lo.d / 4;
    const Raw* yp = reinterpret_cast<const Raw*>(lo.yp) + (int64_t)s * lo.K * n4 + c;
    // Batches of 8 outputs: every load of a batch (indices clamped to K - 1;
    // a clamped re-read is not added) is issued before the adds, which run
    // in k order, in fp32.
    const int K = lo.K;
    float4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int k0 = 0; k0 < K; k0 += 8) {
        Raw v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = yp[(int64_t)min(k0 + u, K - 1) * n4];
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const float4 x = Quad<BF16>::widen(v[u]);
            if (k0 + u == 0) {
                acc = x;
            } else if (k0 + u < K) {
                acc.x = acc.x + x.x;
                acc.y = acc.y + x.y;
                acc.z = acc.z + x.z;
                acc.w = acc.w + x.w;
            }
        }
    }
    reinterpret_cast<float4*>(y + ((int64_t)s * lo.L + l) * lo.d)[c] = acc;
}

// Thread `idx` of the combine grid: four consecutive outputs of one stream.
// Threads past S d / 4 do nothing.  The gated outputs are stored in the
// compute dtype (bf16 or fp32).
__device__ inline void combine_quad(const Layout& lo, int l, float* __restrict__ y, int64_t idx) {
    const int n4 = lo.d / 4;
    if (idx >= (int64_t)lo.S * n4) return;
    const int s = (int)(idx / n4), c = (int)(idx - (int64_t)s * n4);
    if (lo.dtype == 1)
        combine_quad_t<true>(lo, l, y, s, c);
    else
        combine_quad_t<false>(lo, l, y, s, c);
}

// Workgroups of the combine grid: S d / 4 threads, kCombineThreads each.
inline int64_t combine_groups(const Layout& lo) {
    return ((int64_t)lo.S * (lo.d / 4) + kCombineThreads - 1) / kCombineThreads;
}

}  // namespace cmoe
