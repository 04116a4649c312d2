// router.hip - router logits z = W h for the native, Temporal and Spatio
// routers of one layer (Section 2: W^R h; Section 3.2: W^T h; Section 3.3:
// W^S h), all streams at once.
//
// The logits decide expert selection and cache priorities, so they are
// summed in fp64 and rounded to fp32 once (after the bias), like the plain
// definition: the fp32 result then differs from an fp64 sequential sum only
// when that sum lies within ~1e-16 relative of an fp32 rounding boundary.
//
// Work split: one wavefront per 16 experts x 16 streams x one d-chunk
// (split-K), on the fp64 matrix core (v_mfma_f64_16x16x4_f64).  Each split
// stores its 16x16 partial block; the split that finishes last (a per-tile
// counter) adds the blocks in ascending split order, so the result does not
// depend on which split finishes when, and writes the fp32 logits.  Each lane loads 8 consecutive weights (and
// hidden values) at once; the four lane groups of an MFMA take k-slots
// base + 8 g + j for step j, the same permutation for both operands, so every
// product pairs W[e][i] with h[s][i].
#include "cmoe_internal.h"

namespace cmoe {

typedef double f64x4 __attribute__((ext_vector_type(4)));

__device__ inline void load8_as_f64(const void* base, int64_t idx, bool bf16, bool valid, double* out) {
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

// grid: x = n_r * ceil(N/16) * ceil(S/16), z = nsplit; block: 64 (one wavefront)
__global__ __launch_bounds__(64) void router_kernel(Layout lo, int l, const void* h, int dk) {
    const int lane = threadIdx.x;
    const int r16 = lane & 15, g = lane >> 4;
    const int et_n = (lo.N + 15) / 16, st_n = (lo.S + 15) / 16;
    const int tile = blockIdx.x;
    int b = tile;
    const int st = b % st_n;
    b /= st_n;
    const int et = b % et_n;
    const int r = b / et_n;
    const int p = blockIdx.z;
    const int i0 = p * dk;
    const int i1 = min(i0 + dk, lo.d);
    const bool bf16 = lo.dtype == 1;

    const int e_a = et * 16 + r16;  // expert row this lane feeds into A
    const int s_b = st * 16 + r16;  // stream column this lane feeds into B
    const bool va = e_a < lo.N, vb = s_b < lo.S;
    const void* W = r == 0 ? lo.wR : (r == 1 ? lo.wT : lo.wS);
    const int64_t arow = ((int64_t)l * lo.N + (va ? e_a : 0)) * lo.d;
    const int64_t brow = ((int64_t)(vb ? s_b : 0) * lo.L + l) * lo.d;

    f64x4 acc = {0.0, 0.0, 0.0, 0.0};
    for (int base = i0; base < i1; base += 32) {
        double av[8], bv[8];
        load8_as_f64(W, arow + base + 8 * g, bf16, va, av);
        load8_as_f64(h, brow + base + 8 * g, bf16, vb, bv);
#pragma unroll
        for (int j = 0; j < 8; ++j) acc = __builtin_amdgcn_mfma_f64_16x16x4f64(av[j], bv[j], acc, 0, 0, 0);
    }
    // Partial block of this split: value q of lane `lane` at q * 64 + lane.
    double* blk = lo.zpart + ((int64_t)tile * lo.nsplit + p) * 256;
#pragma unroll
    for (int q = 0; q < 4; ++q) blk[q * 64 + lane] = acc[q];

    // The last split to finish adds all splits of the tile in split order,
    // adds the native bias, rounds once and writes the fp32 logits.
    __threadfence();
    unsigned prev = 0;
    if (lane == 0) prev = atomicAdd(&lo.tile_count[tile], 1u);
    prev = __shfl(prev, 0);
    if (prev != (unsigned)(lo.nsplit - 1)) return;
    __threadfence();
    const double* tb = lo.zpart + (int64_t)tile * lo.nsplit * 256;
    double sum[4] = {0.0, 0.0, 0.0, 0.0};
    int q0 = 0;
    for (; q0 + 4 <= lo.nsplit; q0 += 4) {
        double v[4][4];
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
            for (int q = 0; q < 4; ++q) v[u][q] = tb[(q0 + u) * 256 + q * 64 + lane];
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
            for (int q = 0; q < 4; ++q) sum[q] += v[u][q];
    }
    for (; q0 < lo.nsplit; ++q0)
#pragma unroll
        for (int q = 0; q < 4; ++q) sum[q] += tb[q0 * 256 + q * 64 + lane];
    if (lane == 0) lo.tile_count[tile] = 0u;  // ready for the next launch
    // Output of the fp64 16x16x4 MFMA: lane (r16, g) holds D[g + 4 q][r16] in
    // acc[q], i.e. expert row g + 4 q of the tile, stream column r16.
    const int s = st * 16 + r16;
    if (s < lo.S) {
        float* out = lo.logits + (((int64_t)l * lo.S + s) * lo.n_r + r) * lo.N;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = et * 16 + g + 4 * q;
            if (e < lo.N) {
                double z = sum[q];
                if (r == 0 && lo.bias) z += (double)lo.bias[(int64_t)l * lo.N + e];
                out[e] = (float)z;
            }
        }
    }
}

hipError_t launch_router(const Layout& lo, int l, const void* h, hipStream_t st) {
    const int dk = lo.rdk;  // multiple of 32; the last split may be shorter (d % 32 == 0)
    const int tiles = lo.n_r * ((lo.N + 15) / 16) * ((lo.S + 15) / 16);
    hipLaunchKernelGGL(router_kernel, dim3(tiles, 1, lo.nsplit), dim3(64), 0, st, lo, l, h, dk);
    return hipGetLastError();
}

}  // namespace cmoe
