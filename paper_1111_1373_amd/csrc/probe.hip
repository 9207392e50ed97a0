// Streaming copy used to calibrate byte counters and measure reachable HBM bandwidth.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "dtree_probe.h"

namespace {

typedef int i32x4 __attribute__((ext_vector_type(4)));

__global__ void __launch_bounds__(256) copy_kernel(const i32x4 *__restrict__ src,
                                                   i32x4 *__restrict__ dst, int64_t n16) {
    const int64_t stride = int64_t(gridDim.x) * blockDim.x;
    for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n16; i += stride)
        __builtin_nontemporal_store(__builtin_nontemporal_load(src + i), dst + i);
}

}  // namespace

extern "C" dt_status dt_probe_copy(const void *d_src, void *d_dst, int64_t bytes, void *stream) {
    if (bytes < 0 || (bytes & 15) != 0) return DT_ERR_INVALID_ARG;
    if (bytes == 0) return DT_OK;
    if (!d_src || !d_dst) return DT_ERR_INVALID_ARG;
    if (((reinterpret_cast<uintptr_t>(d_src) | reinterpret_cast<uintptr_t>(d_dst)) & 15u) != 0)
        return DT_ERR_INVALID_ARG;
    int dev = 0, n_cu = 0;
    if (hipGetDevice(&dev) != hipSuccess) return DT_ERR_HIP;
    if (hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return DT_ERR_HIP;
    const int64_t n16 = bytes / 16;
    const int64_t want = (n16 + 255) / 256;
    const int64_t blocks = want < int64_t(n_cu) * 8 ? want : int64_t(n_cu) * 8;
    hipLaunchKernelGGL(copy_kernel, dim3(unsigned(blocks)), dim3(256), 0,
                       static_cast<hipStream_t>(stream), static_cast<const i32x4 *>(d_src),
                       static_cast<i32x4 *>(d_dst), n16);
    return hipGetLastError() == hipSuccess ? DT_OK : DT_ERR_HIP;
}
