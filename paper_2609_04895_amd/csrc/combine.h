// combine.h - the gated combine of one layer's expert outputs, as a device
// function: y[s][l] = sum over k of the gated outputs yp[s][k] (the gates are
// already applied by the down projection), added in k order.  Used by the
// stand-alone combine kernel and by the cache-step launch of the next layer,
// which runs it in workgroups of its own.
#pragma once

#include "cmoe_internal.h"

namespace cmoe {

constexpr int kCombineThreads = 256;  // threads per combine workgroup

// Thread `idx` of the combine grid: four consecutive outputs of one stream.
// Threads past S d / 4 do nothing.
__device__ inline void combine_quad(const Layout& lo, int l, float* __restrict__ y, int64_t idx) {
    const int n4 = lo.d / 4;
    if (idx >= (int64_t)lo.S * n4) return;
    const int s = (int)(idx / n4), c = (int)(idx - (int64_t)s * n4);
    const float4* yp = reinterpret_cast<const float4*>(lo.yp) + (int64_t)s * lo.K * n4 + c;
    // Batches of 8 outputs: every load of a batch (indices clamped to K - 1;
    // a clamped re-read is not added) is issued before the adds, which run
    // in k order.
    const int K = lo.K;
    float4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int k0 = 0; k0 < K; k0 += 8) {
        float4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = yp[(int64_t)min(k0 + u, K - 1) * n4];
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            if (k0 + u == 0) {
                acc = v[0];
            } else if (k0 + u < K) {
                acc.x = acc.x + v[u].x;
                acc.y = acc.y + v[u].y;
                acc.z = acc.z + v[u].z;
                acc.w = acc.w + v[u].w;
            }
        }
    }
    reinterpret_cast<float4*>(y + ((int64_t)s * lo.L + l) * lo.d)[c] = acc;
}

// Workgroups of the combine grid: S d / 4 threads, kCombineThreads each.
inline int64_t combine_groups(const Layout& lo) {
    return ((int64_t)lo.S * (lo.d / 4) + kCombineThreads - 1) / kCombineThreads;
}

}  // namespace cmoe
