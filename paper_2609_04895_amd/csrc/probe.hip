// probe.hip - a streaming read of a device buffer with the access pattern of
// the FFN kernels' expert weight loads: 16-byte nontemporal loads, 64 lanes
// covering one contiguous kilobyte per instruction, eight kilobytes in flight
// per wavefront, each wavefront walking its own contiguous block.  Its rate is
// the practical ceiling that the weight stream of one layer step can reach on
// this device, measured in the caller's process.
#include "cmoe_internal.h"

namespace cmoe {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Where the xor of everything read is stored if it equals a value that it
// never takes in practice: the loads are kept, and nothing is written.  (The
// variable has external linkage, so the compiler cannot drop the store, and
// with it the loads.)
__device__ u32x4 g_probe_sink;

namespace {

constexpr int kProbeDepth = 8;  // 1 KB loads in flight per wavefront

// per_wave: 16-byte units of each wavefront's block, a multiple of
// 64 kProbeDepth.
__global__ __launch_bounds__(256) void read_probe_kernel(const u32x4* __restrict__ src, int64_t per_wave) {
    const int lane = threadIdx.x & 63;
    const int64_t wave = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
    const u32x4* p = src + wave * per_wave + lane;
    u32x4 acc = {0u, 0u, 0u, 0u};
    for (int64_t i = 0; i < per_wave; i += 64 * kProbeDepth) {
        u32x4 v[kProbeDepth];
#pragma unroll
        for (int u = 0; u < kProbeDepth; ++u) v[u] = __builtin_nontemporal_load(p + i + 64 * u);
#pragma unroll
        for (int u = 0; u < kProbeDepth; ++u) acc ^= v[u];
    }
    if (acc.x == 0x9E3779B9u && acc.y == 0x7F4A7C15u && acc.z == 0x85EBCA6Bu && acc.w == 0xC2B2AE35u) g_probe_sink = acc;
}

}  // namespace

// 1024 workgroups of four wavefronts (a few per CU on 256 CUs).
constexpr int kProbeBlocks = 1024, kProbeWaves = 4;

int64_t read_probe_units_per_wave(int64_t bytes, int64_t* read_bytes) {
    const int64_t waves = (int64_t)kProbeBlocks * kProbeWaves;
    const int64_t per_wave = bytes / 16 / waves / (64 * kProbeDepth) * (64 * kProbeDepth);
    *read_bytes = per_wave * 16 * waves;
    return per_wave;
}

hipError_t launch_read_probe(const void* src, int64_t per_wave, hipStream_t st, const Timing& tm) {
    launch_kernel(read_probe_kernel, dim3(kProbeBlocks), dim3(64 * kProbeWaves), st, tm,
                  static_cast<const u32x4*>(src), per_wave);
    return hipGetLastError();
}

}  // namespace cmoe
