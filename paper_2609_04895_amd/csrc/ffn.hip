// ffn.hip - the SwiGLU expert FFN over the resident expert weights
// ("execute the MoE layer", Algorithm 2), grouped by expert:
//   a_e = silu(W_gate,e x) * (W_up,e x),  y_(s,k) = g_(s,k) W_down,e a_e,
//   y_s = sum_k y_(s,k)  (k in ascending order).
// Each expert's weights are read once per layer step from its HBM slot,
// whatever the number of tokens routed to it, so the layer step streams
// |union of selected experts| x expert_bytes: the kernels are HBM-bound.
//
// bf16: one wavefront per 16 rows of W_gate and of W_up (gate/up kernel) or
// per 32 rows of W_down (down kernel), on the bf16 matrix core
// (v_mfma_f32_16x16x32_bf16, fp32 accumulation).  The expert's tokens form the
// 16 columns of the B operand (groups of 16 tokens; several groups reuse the
// loaded weights).  Per 64-wide k chunk, lane (r, g) of the A operand holds
// W[row r][kc + 16 g .. + 16]; the two MFMAs of a chunk take k-slots
// kc + 16 g + {0..7} and kc + 16 g + {8..15}, the same for both operands.
// The weights come from the expert's HBM slot in packed order (the fill
// kernel writes it so): each A operand load of a wavefront reads one
// contiguous kilobyte and each wavefront streams one contiguous block.  The
// SwiGLU intermediate is stored in bf16 (the input type of the down kernel's
// matrix core).
//
// fp32: plain VALU kernels, one thread per output row, fp32 accumulation.
#include "cmoe_internal.h"

namespace cmoe {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kNG = 4;   // token groups (of 16) per pass over the weights
constexpr int kUnroll = 4;

__device__ inline bf16x8 as_bf16x8(uint4 v) {
    bf16x8 r;
    __builtin_memcpy(&r, &v, 16);
    return r;
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

// Weights of expert e of layer l in its HBM slot (slot map version sv), or
// nullptr if it has none (cannot happen for a selected expert: the residency
// step maps every member of any cache, and selected experts are members).
__device__ inline const uint16_t* expert_base(const Layout& lo, int l, int sv, int e) {
    const int slot = lo.slot_of[((int64_t)sv * lo.L + l) * lo.N + e];
    if (slot < 0 || slot >= lo.n_slots) return nullptr;
    return reinterpret_cast<const uint16_t*>(lo.arena) + ((int64_t)l * lo.n_slots + slot) * lo.expert_elems;
}

// ---------------------------------------------------------------- bf16
__global__ __launch_bounds__(64) void ffn_up_bf16(Layout lo, int l, int bbuf, int sv, const uint16_t* __restrict__ h) {
    const int ftn = lo.F / 16;
    const int e = blockIdx.x / ftn, ft = blockIdx.x - e * ftn;
    const int m = lo.bcount[(int64_t)bbuf * lo.N + e];
    if (m == 0) return;
    const int32_t* bk = lo.pairs + ((int64_t)bbuf * lo.N + e) * lo.S;
    const uint16_t* Wg = expert_base(lo, l, sv, e);
    if (!Wg) return;
    const int lane = threadIdx.x, r = lane & 15, g = lane >> 4;
    // packed slot layout: chunk c of this row tile is 256 units of 16 bytes,
    // gate half 0, gate half 1, up half 0, up half 1, each 64 units
    const uint4* tileA = reinterpret_cast<const uint4*>(Wg) + (int64_t)ft * (lo.d / 64) * 256 + lane;
    uint16_t* act = reinterpret_cast<uint16_t*>(lo.act);
    const int d = lo.d;
    const int nchunk = d / 64;

    for (int t0 = 0; t0 < m; t0 += 16 * kNG) {
        const int ng = min(kNG, (m - t0 + 15) / 16);
        const uint16_t* xb[kNG];
        bool xv[kNG];
#pragma unroll
        for (int q = 0; q < kNG; ++q) {
            const int tok = t0 + 16 * q + r;
            xv[q] = q < ng && tok < m;
            const int s = xv[q] ? (bk[tok] >> 8) : 0;
            xb[q] = h + ((int64_t)s * lo.L + l) * d + 16 * g;
        }
        f32x4 cg[kNG], cu[kNG];
#pragma unroll
        for (int q = 0; q < kNG; ++q) {
            cg[q] = f32x4{0.f, 0.f, 0.f, 0.f};
            cu[q] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
        int c = 0;
        for (; c + kUnroll <= nchunk; c += kUnroll) {
            uint4 G[kUnroll][2], U[kUnroll][2];
#pragma unroll
            for (int i = 0; i < kUnroll; ++i) {
                const uint4* ch = tileA + (int64_t)(c + i) * 256;
                G[i][0] = ch[0];
                G[i][1] = ch[64];
                U[i][0] = ch[128];
                U[i][1] = ch[192];
            }
#pragma unroll
            for (int q = 0; q < kNG; ++q) {
                if (q >= ng) break;
#pragma unroll
                for (int i = 0; i < kUnroll; ++i) {
                    const int kc = (c + i) * 64;
                    uint4 x0 = {0, 0, 0, 0}, x1 = {0, 0, 0, 0};
                    if (xv[q]) {
                        x0 = *reinterpret_cast<const uint4*>(xb[q] + kc);
                        x1 = *reinterpret_cast<const uint4*>(xb[q] + kc + 8);
                    }
                    cg[q] = mfma_bf16(G[i][0], x0, cg[q]);
                    cg[q] = mfma_bf16(G[i][1], x1, cg[q]);
                    cu[q] = mfma_bf16(U[i][0], x0, cu[q]);
                    cu[q] = mfma_bf16(U[i][1], x1, cu[q]);
                }
            }
        }
        for (; c < nchunk; ++c) {
            const int kc = c * 64;
            const uint4* ch = tileA + (int64_t)c * 256;
            const uint4 g0 = ch[0];
            const uint4 g1 = ch[64];
            const uint4 u0 = ch[128];
            const uint4 u1 = ch[192];
#pragma unroll
            for (int q = 0; q < kNG; ++q) {
                if (q >= ng) break;
                uint4 x0 = {0, 0, 0, 0}, x1 = {0, 0, 0, 0};
                if (xv[q]) {
                    x0 = *reinterpret_cast<const uint4*>(xb[q] + kc);
                    x1 = *reinterpret_cast<const uint4*>(xb[q] + kc + 8);
                }
                cg[q] = mfma_bf16(g0, x0, cg[q]);
                cg[q] = mfma_bf16(g1, x1, cg[q]);
                cu[q] = mfma_bf16(u0, x0, cu[q]);
                cu[q] = mfma_bf16(u1, x1, cu[q]);
            }
        }
        // D[i][j]: row i = 4 g + rr of this 16-row tile, token column j = r
#pragma unroll
        for (int q = 0; q < kNG; ++q) {
            if (q >= ng) break;
            const int tok = t0 + 16 * q + r;
            if (tok < m) {
                uint2 o;
                o.x = pack_bf16x2(silu_mul(cg[q][0], cu[q][0]), silu_mul(cg[q][1], cu[q][1]));
                o.y = pack_bf16x2(silu_mul(cg[q][2], cu[q][2]), silu_mul(cg[q][3], cu[q][3]));
                const int pair = bk[tok];
                const int64_t row = (int64_t)(pair >> 8) * lo.K + (pair & 255);  // token (s, k)
                *reinterpret_cast<uint2*>(act + row * lo.F + ft * 16 + 4 * g) = o;
            }
        }
    }
}

__global__ __launch_bounds__(64) void ffn_down_bf16(Layout lo, int l, int bbuf, int sv) {
    const int dtn = lo.d / 32;
    const int e = blockIdx.x / dtn, dt = blockIdx.x - e * dtn;
    const int m = lo.bcount[(int64_t)bbuf * lo.N + e];
    if (m == 0) return;
    const int32_t* bk = lo.pairs + ((int64_t)bbuf * lo.N + e) * lo.S;
    const int F = lo.F;
    const uint16_t* Wbase = expert_base(lo, l, sv, e);
    if (!Wbase) return;
    const int lane = threadIdx.x, r = lane & 15, g = lane >> 4;
    // packed slot layout: after the gate/up part (F d / 4 units), chunk c of
    // this 32-row tile is 256 units: rows 0-15 half 0, half 1, rows 16-31
    // half 0, half 1, each 64 units
    const uint4* tileB =
        reinterpret_cast<const uint4*>(Wbase) + (int64_t)F * lo.d / 4 + (int64_t)dt * (F / 64) * 256 + lane;
    const uint16_t* act = reinterpret_cast<const uint16_t*>(lo.act);
    const int nchunk = F / 64;

    for (int t0 = 0; t0 < m; t0 += 16 * kNG) {
        const int ng = min(kNG, (m - t0 + 15) / 16);
        const uint16_t* xb[kNG];
        bool xv[kNG];
#pragma unroll
        for (int q = 0; q < kNG; ++q) {
            const int tok = t0 + 16 * q + r;
            xv[q] = q < ng && tok < m;
            const int pair = xv[q] ? bk[tok] : 0;
            xb[q] = act + ((int64_t)(pair >> 8) * lo.K + (pair & 255)) * F + 16 * g;
        }
        f32x4 c0[kNG], c1[kNG];
#pragma unroll
        for (int q = 0; q < kNG; ++q) {
            c0[q] = f32x4{0.f, 0.f, 0.f, 0.f};
            c1[q] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
        int c = 0;
        for (; c + kUnroll <= nchunk; c += kUnroll) {
            uint4 A0[kUnroll][2], A1[kUnroll][2];
#pragma unroll
            for (int i = 0; i < kUnroll; ++i) {
                const uint4* ch = tileB + (int64_t)(c + i) * 256;
                A0[i][0] = ch[0];
                A0[i][1] = ch[64];
                A1[i][0] = ch[128];
                A1[i][1] = ch[192];
            }
#pragma unroll
            for (int q = 0; q < kNG; ++q) {
                if (q >= ng) break;
#pragma unroll
                for (int i = 0; i < kUnroll; ++i) {
                    const int kc = (c + i) * 64;
                    uint4 x0 = {0, 0, 0, 0}, x1 = {0, 0, 0, 0};
                    if (xv[q]) {
                        x0 = *reinterpret_cast<const uint4*>(xb[q] + kc);
                        x1 = *reinterpret_cast<const uint4*>(xb[q] + kc + 8);
                    }
                    c0[q] = mfma_bf16(A0[i][0], x0, c0[q]);
                    c0[q] = mfma_bf16(A0[i][1], x1, c0[q]);
                    c1[q] = mfma_bf16(A1[i][0], x0, c1[q]);
                    c1[q] = mfma_bf16(A1[i][1], x1, c1[q]);
                }
            }
        }
        for (; c < nchunk; ++c) {
            const int kc = c * 64;
            const uint4* ch = tileB + (int64_t)c * 256;
            const uint4 p0 = ch[0];
            const uint4 p1 = ch[64];
            const uint4 q0 = ch[128];
            const uint4 q1 = ch[192];
#pragma unroll
            for (int q = 0; q < kNG; ++q) {
                if (q >= ng) break;
                uint4 x0 = {0, 0, 0, 0}, x1 = {0, 0, 0, 0};
                if (xv[q]) {
                    x0 = *reinterpret_cast<const uint4*>(xb[q] + kc);
                    x1 = *reinterpret_cast<const uint4*>(xb[q] + kc + 8);
                }
                c0[q] = mfma_bf16(p0, x0, c0[q]);
                c0[q] = mfma_bf16(p1, x1, c0[q]);
                c1[q] = mfma_bf16(q0, x0, c1[q]);
                c1[q] = mfma_bf16(q1, x1, c1[q]);
            }
        }
#pragma unroll
        for (int q = 0; q < kNG; ++q) {
            if (q >= ng) break;
            const int tok = t0 + 16 * q + r;
            if (tok < m) {
                const int pair = bk[tok];
                const int s = pair >> 8, k = pair & 255;
                const float gk = lo.gates[((int64_t)l * lo.S + s) * lo.K + k];
                float* dst = lo.yp + ((int64_t)s * lo.K + k) * lo.d + dt * 32 + 4 * g;
                *reinterpret_cast<float4*>(dst) = make_float4(gk * c0[q][0], gk * c0[q][1], gk * c0[q][2], gk * c0[q][3]);
                *reinterpret_cast<float4*>(dst + 16) =
                    make_float4(gk * c1[q][0], gk * c1[q][1], gk * c1[q][2], gk * c1[q][3]);
            }
        }
    }
}

// ---------------------------------------------------------------- fp32
__global__ __launch_bounds__(64) void ffn_up_f32(Layout lo, int l, int bbuf, int sv, const float* __restrict__ h) {
    const int ftn = lo.F / 64;
    const int e = blockIdx.x / ftn, ft = blockIdx.x - e * ftn;
    const int m = lo.bcount[(int64_t)bbuf * lo.N + e];
    if (m == 0) return;
    const int32_t* bk = lo.pairs + ((int64_t)bbuf * lo.N + e) * lo.S;
    const int slot = lo.slot_of[((int64_t)sv * lo.L + l) * lo.N + e];
    if (slot < 0 || slot >= lo.n_slots) return;
    const float* Wg = reinterpret_cast<const float*>(lo.arena) + ((int64_t)l * lo.n_slots + slot) * lo.expert_elems;
    const float* Wu = Wg + (int64_t)lo.F * lo.d;
    const int f = ft * 64 + threadIdx.x;
    float* act = reinterpret_cast<float*>(lo.act);
    for (int tok = 0; tok < m; ++tok) {
        const int pair = bk[tok];
        const int s = pair >> 8;
        const float* x = h + ((int64_t)s * lo.L + l) * lo.d;
        float ag = 0.0f, au = 0.0f;
        for (int i = 0; i < lo.d; ++i) {
            ag = __builtin_fmaf(Wg[(int64_t)f * lo.d + i], x[i], ag);
            au = __builtin_fmaf(Wu[(int64_t)f * lo.d + i], x[i], au);
        }
        act[((int64_t)s * lo.K + (pair & 255)) * lo.F + f] = ag / (1.0f + expf(-ag)) * au;
    }
}

__global__ __launch_bounds__(64) void ffn_down_f32(Layout lo, int l, int bbuf, int sv) {
    const int dtn = lo.d / 64;
    const int e = blockIdx.x / dtn, dt = blockIdx.x - e * dtn;
    const int m = lo.bcount[(int64_t)bbuf * lo.N + e];
    if (m == 0) return;
    const int32_t* bk = lo.pairs + ((int64_t)bbuf * lo.N + e) * lo.S;
    const int slot = lo.slot_of[((int64_t)sv * lo.L + l) * lo.N + e];
    if (slot < 0 || slot >= lo.n_slots) return;
    const float* Wd = reinterpret_cast<const float*>(lo.arena) + ((int64_t)l * lo.n_slots + slot) * lo.expert_elems +
                      2 * (int64_t)lo.F * lo.d;
    const int j = dt * 64 + threadIdx.x;
    const float* act = reinterpret_cast<const float*>(lo.act);
    for (int tok = 0; tok < m; ++tok) {
        const int pair = bk[tok];
        const int s = pair >> 8, k = pair & 255;
        const float* av = act + ((int64_t)s * lo.K + k) * lo.F;
        float acc = 0.0f;
        for (int f = 0; f < lo.F; ++f) acc = __builtin_fmaf(Wd[(int64_t)j * lo.F + f], av[f], acc);
        const float gk = lo.gates[((int64_t)l * lo.S + s) * lo.K + k];
        lo.yp[((int64_t)s * lo.K + k) * lo.d + j] = gk * acc;
    }
}

// ---------------------------------------------------------------- combine
__global__ __launch_bounds__(64) void combine_kernel(Layout lo, int l, float* __restrict__ y) {
    const int n4 = lo.d / 4;
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= (int64_t)lo.S * n4) return;
    const int s = (int)(idx / n4), c = (int)(idx - (int64_t)s * n4);
    const float4* yp = reinterpret_cast<const float4*>(lo.yp) + (int64_t)s * lo.K * n4 + c;
    float4 acc = yp[0];
    int k = 1;
    for (; k + 8 <= lo.K; k += 8) {  // loads first, then the adds in k order
        float4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = yp[(int64_t)(k + u) * n4];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            acc.x = acc.x + v[u].x;
            acc.y = acc.y + v[u].y;
            acc.z = acc.z + v[u].z;
            acc.w = acc.w + v[u].w;
        }
    }
    for (; k < lo.K; ++k) {
        const float4 v = yp[(int64_t)k * n4];
        acc.x = acc.x + v.x;
        acc.y = acc.y + v.y;
        acc.z = acc.z + v.z;
        acc.w = acc.w + v.w;
    }
    reinterpret_cast<float4*>(y + ((int64_t)s * lo.L + l) * lo.d)[c] = acc;
}

}  // namespace

hipError_t launch_ffn_up(const Layout& lo, int l, int bbuf, int sv, const void* h, hipStream_t st) {
    if (lo.dtype == 1)
        hipLaunchKernelGGL(ffn_up_bf16, dim3(lo.N * (lo.F / 16)), dim3(64), 0, st, lo, l, bbuf, sv,
                           static_cast<const uint16_t*>(h));
    else
        hipLaunchKernelGGL(ffn_up_f32, dim3(lo.N * (lo.F / 64)), dim3(64), 0, st, lo, l, bbuf, sv,
                           static_cast<const float*>(h));
    return hipGetLastError();
}

hipError_t launch_ffn_down(const Layout& lo, int l, int bbuf, int sv, hipStream_t st) {
    if (lo.dtype == 1)
        hipLaunchKernelGGL(ffn_down_bf16, dim3(lo.N * (lo.d / 32)), dim3(64), 0, st, lo, l, bbuf, sv);
    else
        hipLaunchKernelGGL(ffn_down_f32, dim3(lo.N * (lo.d / 64)), dim3(64), 0, st, lo, l, bbuf, sv);
    return hipGetLastError();
}

hipError_t launch_combine(const Layout& lo, int l, float* y, hipStream_t st) {
    const int64_t n = (int64_t)lo.S * (lo.d / 4);
    hipLaunchKernelGGL(combine_kernel, dim3((unsigned)((n + 63) / 64)), dim3(64), 0, st, lo, l, y);
    return hipGetLastError();
}

}  // namespace cmoe
