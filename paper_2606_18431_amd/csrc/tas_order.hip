// tas_order.hip - the launch order of the next simulation pass.
//
// Instances are independent and their results do not depend on when they
// run, but a launch lasts until its slowest workgroup ends: started last, a
// long instance leaves most of the chip idle at the end. The next launch
// therefore starts the instances with the most work first (longest
// processing time first). The work key counts the loop steps an instance's
// wave ran in the previous launch, weighted by their cost (iterations,
// formation passes, emission chunks), which the simulation kernel records.
// Its wall-clock time is a worse key: the waves that share a SIMD do not
// issue equally (older waves win arbitration), so a duration says as much
// about the slot an instance had as about its work. With as many instances
// as resident slots the order only decides that arbitration, and the step
// count still ranks the long instances first. One workgroup sorts up to
// kMaxOrdered (work, index) pairs in LDS with a bitonic network.
#include <hip/hip_runtime.h>

#include "tas_internal.h"

namespace tas {
namespace {

constexpr int kOrderThreads = 1024;

__global__ __launch_bounds__(kOrderThreads) void order_kernel(const int64_t *work, int32_t *order,
                                                              int32_t n, int32_t n2) {
    extern __shared__ __align__(16) unsigned char smem[];
    uint64_t *key = (uint64_t *)smem;
    // ascending keys: the most work first, ties by index
    for (int i = (int)threadIdx.x; i < n2; i += kOrderThreads) {
        uint64_t k = ~0ull;
        if (i < n) {
            const int64_t d = work[i] < 0 ? 0 : (work[i] > (int64_t(1) << 39) ? int64_t(1) << 39 : work[i]);
            k = ((uint64_t)((int64_t(1) << 39) - d) << 24) | (uint64_t)i;
        }
        key[i] = k;
    }
    __syncthreads();
    for (int size = 2; size <= n2; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int i = (int)threadIdx.x; i < n2; i += kOrderThreads) {
                const int j = i ^ stride;
                if (j > i) {
                    const uint64_t x = key[i], y = key[j];
                    const bool up = (i & size) == 0;
                    if ((x > y) == up) key[i] = y, key[j] = x;
                }
            }
            __syncthreads();
        }
    }
    for (int i = (int)threadIdx.x; i < n; i += kOrderThreads)
        order[i] = (int32_t)(key[i] & 0xFFFFFFu);
}

}  // namespace
}  // namespace tas

int tas_launch_order(const int64_t *work, int32_t *order, int32_t n, void *stream) {
    if (n <= 1 || n > tas::kMaxOrdered) return 0;
    int32_t n2 = 1;
    while (n2 < n) n2 <<= 1;
    const size_t lds = (size_t)n2 * 8;
    if (lds > 65536 && hipFuncSetAttribute((const void *)tas::order_kernel,
                                           hipFuncAttributeMaxDynamicSharedMemorySize,
                                           (int)lds) != hipSuccess)
        return -4;
    hipLaunchKernelGGL(tas::order_kernel, dim3(1), dim3(tas::kOrderThreads), lds,
                       (hipStream_t)stream, work, order, n, n2);
    return hipGetLastError() == hipSuccess ? 0 : -4;
}
