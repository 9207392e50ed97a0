// Streaming copy and streaming read: calibrate byte counters and measure the HBM bandwidth a
// plain kernel reaches on this device.
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

// Read-only stream: each wavefront reads 16 KiB tiles (16 vectors per lane, coalesced),
// grid-strided.  The values are folded into one word that is stored only if it equals a
// constant no input of this library produces, so the loads cannot be dropped and nothing
// is written in practice.
__global__ void __launch_bounds__(512) read_kernel(const i32x4 *__restrict__ src, int64_t n16,
                                                   int32_t *__restrict__ sink) {
    const int lane = threadIdx.x & 63;
    const int64_t waves = int64_t(gridDim.x) * (blockDim.x >> 6);
    const int64_t n_tiles = n16 / 1024;
    int32_t acc = 0;
    for (int64_t t = int64_t(blockIdx.x) * (blockDim.x >> 6) + (threadIdx.x >> 6); t < n_tiles;
         t += waves) {
        i32x4 v[16];
#pragma unroll
        for (int k = 0; k < 16; ++k) v[k] = __builtin_nontemporal_load(src + t * 1024 + k * 64 + lane);
#pragma unroll
        for (int k = 0; k < 16; ++k) acc ^= v[k].x ^ v[k].y ^ v[k].z ^ v[k].w;
    }
    // the tail past the last whole tile
    const int64_t gid = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    for (int64_t i = n_tiles * 1024 + gid; i < n16; i += int64_t(gridDim.x) * blockDim.x) {
        const i32x4 v = __builtin_nontemporal_load(src + i);
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    if (acc == int32_t(0x5EEDF00D) && gid == 0x7FFFFFFF) sink[0] = acc;
}

}  // namespace

extern "C" dt_status dt_probe_read(const void *d_src, int64_t bytes, int32_t *d_sink,
                                   int32_t waves_per_cu, void *stream) {
    if (bytes < 0 || (bytes & 15) != 0) return DT_ERR_INVALID_ARG;
    if (waves_per_cu < 1 || waves_per_cu > 32) return DT_ERR_INVALID_ARG;
    if (bytes == 0) return DT_OK;
    if (!d_src || !d_sink || (reinterpret_cast<uintptr_t>(d_src) & 15u) != 0)
        return DT_ERR_INVALID_ARG;
    int dev = 0, n_cu = 0;
    if (hipGetDevice(&dev) != hipSuccess) return DT_ERR_HIP;
    if (hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return DT_ERR_HIP;
    const int waves = waves_per_cu < 8 ? waves_per_cu : 8;            // per workgroup
    const int64_t blocks = int64_t(n_cu) * ((waves_per_cu + waves - 1) / waves);
    hipLaunchKernelGGL(read_kernel, dim3(unsigned(blocks)), dim3(unsigned(waves * 64)), 0,
                       static_cast<hipStream_t>(stream), static_cast<const i32x4 *>(d_src),
                       bytes / 16, d_sink);
    return hipGetLastError() == hipSuccess ? DT_OK : DT_ERR_HIP;
}

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
