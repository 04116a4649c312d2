// combine.hip - stand-alone launch of the gated combine of a layer's expert
// outputs (the device function is in combine.h).  A token step launches it
// for its last layer only: the combine of every other layer runs in the
// cache-step launch of the layer after it, which does not depend on it.
#include "combine.h"

namespace cmoe {

namespace {

__global__ __launch_bounds__(kCombineThreads) void combine_kernel(Layout lo, int l, float* __restrict__ y) {
    combine_quad(lo, l, y, (int64_t)blockIdx.x * kCombineThreads + threadIdx.x);
}

}  // namespace

hipError_t launch_combine(const Layout& lo, int l, float* y, hipStream_t st, const Timing& tm) {
    launch_kernel(combine_kernel, dim3((unsigned)combine_groups(lo)), dim3(kCombineThreads), st, tm, lo, l, y);
    return hipGetLastError();
}

}  // namespace cmoe
