// fill.hip - copies newly resident experts from the cold pool into their HBM
// slots (the demand loads and proactive loads of Section 2 / Algorithm 2, as
// physical transfers).  The list of (expert, slot) pairs and its length are
// produced on the device by the residency step, so the copy is a kernel that
// reads the list rather than host-issued memcpys: no host synchronisation per
// layer.  With an empty list it returns at once.  The pool may be pinned host
// memory mapped into the device; the copy then runs over the host link.
#include "cmoe_internal.h"

namespace cmoe {

namespace {

__global__ __launch_bounds__(256) void fill_kernel(Layout lo, int l, int kind) {
    const int n = lo.fill_count[l * 2 + kind];
    if (n == 0) return;
    const int64_t bytes = lo.expert_elems * (lo.dtype == 1 ? 2 : 4);
    const int64_t n16 = bytes / 16;
    const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t gs = (int64_t)gridDim.x * blockDim.x;
    const int32_t* fl = lo.fill_list + ((int64_t)l * 2 + kind) * lo.N * 2;
    for (int f = 0; f < n; ++f) {
        const int e = fl[2 * f], q = fl[2 * f + 1];
        const uint4* src =
            reinterpret_cast<const uint4*>(static_cast<const char*>(lo.pool) + ((int64_t)l * lo.N + e) * bytes);
        uint4* dst = reinterpret_cast<uint4*>(static_cast<char*>(lo.arena) + ((int64_t)l * lo.n_slots + q) * bytes);
        for (int64_t i = gid; i < n16; i += gs) dst[i] = src[i];
    }
}

}  // namespace

hipError_t launch_fill(const Layout& lo, int l, int kind, hipStream_t st) {
    hipLaunchKernelGGL(fill_kernel, dim3(512), dim3(256), 0, st, lo, l, kind);
    return hipGetLastError();
}

}  // namespace cmoe
