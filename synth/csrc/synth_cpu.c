/*
 * synth_cpu.c - host twin of the seeded synthetic-input generator.
 *
 * This module produces the inputs of the cache-aware MoE decode step (router
 * weights, expert weights, AR(1) hidden states).  It holds none of the
 * method's arithmetic.  The same generator is implemented a second time, on
 * the GPU, in synth_hip.hip; both follow the definition below and must give
 * bit-identical tensors (checked by FNV-1a checksums in the GPU tests).
 *
 * Definition
 *   SplitMix64 (Steele, Lea & Flood, "Fast splittable pseudorandom number
 *   generators", OOPSLA 2014): golden-ratio increment GAMMA and the output
 *   mixing function mix().
 *   key(seed, tid)   = mix(seed XOR mix(tid + GAMMA))
 *   draw(key, i)     = mix(key + (i + 1) * GAMMA)          (mod 2^64)
 *   normal(key, i)   = n = sum_{j<4} ((draw >> 16j) & 0xFFFF) - 131070
 *                      (Irwin-Hall sum of four 16-bit uniforms, centred;
 *                      variance 65536^2/3, support +-3.46 sigma)
 *   value            = (float)((double)n * scale), scale = sigma*sqrt(3)/65536
 *                      computed once on the host in double and passed in.
 *   bf16 storage     = round-to-nearest-even of the fp32 bit pattern.
 *   AR(1) hidden     = h_0 = fl32(e_0 * c0), c0 = fl32(1/sqrt(1-rho^2));
 *                      h_t = fl32(fl32(rho * h_{t-1}) + e_t)   (no contraction)
 *                      with e_t = normal(key_h, t*d + j) at unit sigma.
 *
 * Build with -ffp-contract=off so that rho*h + e is never fused.
 */
#include <stdint.h>
#include <string.h>

#define SYN_GAMMA 0x9E3779B97F4A7C15ULL

static inline uint64_t syn_mix(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

uint64_t syn_key(uint64_t seed, uint64_t tid) {
    return syn_mix(seed ^ syn_mix(tid + SYN_GAMMA));
}

uint64_t syn_draw(uint64_t key, uint64_t i) {
    return syn_mix(key + (i + 1ULL) * SYN_GAMMA);
}

static inline float syn_normal(uint64_t key, uint64_t i, double scale) {
    uint64_t r = syn_mix(key + (i + 1ULL) * SYN_GAMMA);
    int64_t n = (int64_t)(r & 0xFFFFULL) + (int64_t)((r >> 16) & 0xFFFFULL) +
                (int64_t)((r >> 32) & 0xFFFFULL) + (int64_t)((r >> 48) & 0xFFFFULL) - 131070;
    return (float)((double)n * scale);
}

static inline uint16_t syn_bf16_bits(float x) {
    uint32_t u;
    memcpy(&u, &x, 4);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

static inline float syn_bf16_to_f32(uint16_t b) {
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, 4);
    return f;
}

/* n normal values starting at element index `first` of tensor `key`.
 * If round_bf16 != 0 the values are rounded to bf16 and widened back, so the
 * fp32 output equals what a bf16 tensor stores. */
void syn_normal_f32(uint64_t key, uint64_t first, int64_t n, double scale,
                    int round_bf16, float* out) {
    for (int64_t i = 0; i < n; ++i) {
        float v = syn_normal(key, first + (uint64_t)i, scale);
        out[i] = round_bf16 ? syn_bf16_to_f32(syn_bf16_bits(v)) : v;
    }
}

/* Same values stored as raw bf16 bit patterns. */
void syn_normal_bf16(uint64_t key, uint64_t first, int64_t n, double scale, uint16_t* out) {
    for (int64_t i = 0; i < n; ++i) out[i] = syn_bf16_bits(syn_normal(key, first + (uint64_t)i, scale));
}

/* AR(1) hidden states of one (stream, layer): out[t][d] for t < T.
 * The recurrence runs on the fp32 values; the stored value is optionally
 * rounded to bf16 (then widened) as a bf16 tensor would hold it. */
void syn_ar1_f32(uint64_t key, int32_t T, int32_t d, float rho, float c0, double scale,
                 int round_bf16, float* out) {
    for (int32_t j = 0; j < d; ++j) {
        float h = 0.0f;
        for (int32_t t = 0; t < T; ++t) {
            float e = syn_normal(key, (uint64_t)t * (uint64_t)d + (uint64_t)j, scale);
            if (t == 0) {
                h = e * c0;
            } else {
                volatile float rh = rho * h; /* one rounding, then the add */
                h = rh + e;
            }
            out[(int64_t)t * d + j] = round_bf16 ? syn_bf16_to_f32(syn_bf16_bits(h)) : h;
        }
    }
}

/* 64-bit FNV-1a over a byte buffer (Fowler, Noll, Vo). */
uint64_t syn_fnv1a(const void* data, int64_t nbytes, uint64_t h) {
    const unsigned char* p = (const unsigned char*)data;
    for (int64_t i = 0; i < nbytes; ++i) {
        h ^= (uint64_t)p[i];
        h *= 0x100000001B3ULL;
    }
    return h;
}
