// synth_hip.hip - device twin of the seeded synthetic-input generator.
//
// Same definition as synth_cpu.c (SplitMix64 counter-based draws, centred
// Irwin-Hall sum of four 16-bit uniforms, fp64 scaling, bf16 round-to-nearest-
// even, AR(1) recurrence in fp32 without contraction).  It fills device (or
// host-mapped) memory so that the multi-GB inputs of the large workloads never
// pass through the host.  It holds none of the method's arithmetic.
//
// Build with -ffp-contract=off.
#include <hip/hip_runtime.h>
#include <stdint.h>

#define SYN_GAMMA 0x9E3779B97F4A7C15ULL

__device__ __host__ static inline uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

__device__ __host__ static inline uint64_t key_of(uint64_t seed, uint64_t tid) {
    return mix64(seed ^ mix64(tid + SYN_GAMMA));
}

__device__ static inline float normal_at(uint64_t key, uint64_t i, double scale) {
    uint64_t r = mix64(key + (i + 1ULL) * SYN_GAMMA);
    int64_t n = (int64_t)(r & 0xFFFFULL) + (int64_t)((r >> 16) & 0xFFFFULL) +
                (int64_t)((r >> 32) & 0xFFFFULL) + (int64_t)((r >> 48) & 0xFFFFULL) - 131070;
    return (float)((double)n * scale);
}

__device__ static inline uint16_t bf16_bits(float x) {
    uint32_t u = __float_as_uint(x);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// A batch of tensors: tensor b (b < nb) has id tid0 + b * tid_stride, holds
// `per` elements and is written at out + b * per.  One grid row per tensor.
__global__ void syn_fill_kernel(uint64_t seed, uint64_t tid0, uint64_t tid_stride, int64_t per,
                                double scale, int bf16, void* out) {
    const uint64_t b = blockIdx.y;
    const uint64_t key = key_of(seed, tid0 + b * tid_stride);
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < per; i += stride) {
        float v = normal_at(key, (uint64_t)i, scale);
        if (bf16)
            ((uint16_t*)out)[b * per + i] = bf16_bits(v);
        else
            ((float*)out)[b * per + i] = v;
    }
}

// AR(1) hidden states, written token-major: out[t][s][l][j] for all streams s
// < S and layers l < L.  One thread per (s, l, j).  Key of (s, l) is
// key_of(seed, tid0 + s * tid_s + l * tid_l).
__global__ void syn_ar1_kernel(uint64_t seed, uint64_t tid0, uint64_t tid_s, uint64_t tid_l,
                               int32_t S, int32_t L, int32_t d, int32_t T, float rho, float c0,
                               double scale, int bf16, void* out) {
    const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t per_tok = (int64_t)S * L * d;
    if (g >= per_tok) return;
    const int32_t j = (int32_t)(g % d);
    const int32_t l = (int32_t)((g / d) % L);
    const int32_t s = (int32_t)(g / ((int64_t)d * L));
    const uint64_t key = key_of(seed, tid0 + (uint64_t)s * tid_s + (uint64_t)l * tid_l);
    float h = 0.0f;
    for (int32_t t = 0; t < T; ++t) {
        float e = normal_at(key, (uint64_t)t * (uint64_t)d + (uint64_t)j, scale);
        if (t == 0) {
            h = __fmul_rn(e, c0);
        } else {
            h = __fadd_rn(__fmul_rn(rho, h), e);
        }
        const int64_t o = (int64_t)t * per_tok + g;
        if (bf16)
            ((uint16_t*)out)[o] = bf16_bits(h);
        else
            ((float*)out)[o] = h;
    }
}

extern "C" {

// Fills nb tensors of `per` elements each (see syn_fill_kernel).  Returns a
// hipError_t value (0 = success).
int syn_dev_fill(uint64_t seed, uint64_t tid0, uint64_t tid_stride, int64_t nb, int64_t per,
                 double scale, int bf16, void* out, void* stream) {
    if (nb <= 0 || per <= 0) return 0;
    int64_t bx = (per + 255) / 256;
    if (bx > 4096) bx = 4096;
    const int64_t esz = bf16 ? 2 : 4;
    for (int64_t b0 = 0; b0 < nb; b0 += 65535) {  // grid.y holds at most 65535 tensors
        const int64_t nbc = (nb - b0 < 65535) ? (nb - b0) : 65535;
        hipLaunchKernelGGL(syn_fill_kernel, dim3((unsigned)bx, (unsigned)nbc, 1), dim3(256), 0,
                           (hipStream_t)stream, seed, tid0 + (uint64_t)b0 * tid_stride, tid_stride, per,
                           scale, bf16, (void*)((char*)out + b0 * per * esz));
        int rc = (int)hipGetLastError();
        if (rc) return rc;
    }
    return 0;
}

int syn_dev_ar1(uint64_t seed, uint64_t tid0, uint64_t tid_s, uint64_t tid_l, int32_t S, int32_t L,
                int32_t d, int32_t T, float rho, float c0, double scale, int bf16, void* out,
                void* stream) {
    const int64_t n = (int64_t)S * L * d;
    if (n <= 0 || T <= 0) return 0;
    hipLaunchKernelGGL(syn_ar1_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0,
                       (hipStream_t)stream, seed, tid0, tid_s, tid_l, S, L, d, T, rho, c0, scale, bf16,
                       out);
    return (int)hipGetLastError();
}

// Pinned, device-mapped host memory of exactly `bytes` bytes (a cold pool in
// host memory), or NULL.  Returns a hipError_t value.
int syn_host_alloc(int64_t bytes, void** out) {
    *out = nullptr;
    const hipError_t e = hipHostMalloc(out, (size_t)bytes, hipHostMallocDefault);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        *out = nullptr;
    }
    return (int)e;
}

int syn_host_free(void* p) { return p ? (int)hipHostFree(p) : 0; }

}  // extern "C"
