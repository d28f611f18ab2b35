// Streaming copy and read kernels of known traffic, used by the benchmark as
// the measured HBM ceilings of this GPU (read only; read + write) and as the
// reference kernel that scales the rocprofv3 FETCH_SIZE / WRITE_SIZE
// counters to bytes.  Not part of the routing ABI.
#include <hip/hip_runtime.h>

typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));

__global__ void __launch_bounds__(256)
hbm_probe_copy16(const u32x4_t *__restrict__ src, u32x4_t *__restrict__ dst, long long n)
{
    const long long stride = (long long)gridDim.x * 256;
    for (long long i = (long long)blockIdx.x * 256 + threadIdx.x; i < n; i += stride)
        __builtin_nontemporal_store(__builtin_nontemporal_load(src + i), dst + i);
}

__global__ void __launch_bounds__(256)
hbm_probe_read16(const u32x4_t *__restrict__ src, unsigned *__restrict__ sink, long long n)
{
    const long long stride = (long long)gridDim.x * 256;
    unsigned acc = 0;
    for (long long i = (long long)blockIdx.x * 256 + threadIdx.x; i < n; i += stride) {
        const u32x4_t v = __builtin_nontemporal_load(src + i);
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    if (acc == 0x9e3779b9u)  // keeps the loads; practically never true
        sink[0] = acc;
}

// bytes must be a multiple of 16 and both pointers 16-byte aligned.
extern "C" int hbm_probe_copy(const void *src, void *dst, long long bytes, int blocks,
                              void *stream)
{
    if (bytes % 16 || blocks < 1 || (reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst)) % 16)
        return -1;
    hipLaunchKernelGGL(hbm_probe_copy16, dim3(blocks), dim3(256), 0,
                       static_cast<hipStream_t>(stream), static_cast<const u32x4_t *>(src),
                       static_cast<u32x4_t *>(dst), bytes / 16);
    return hipGetLastError() == hipSuccess ? 0 : -2;
}

extern "C" int hbm_probe_read(const void *src, void *sink, long long bytes, int blocks,
                              void *stream)
{
    if (bytes % 16 || blocks < 1 || reinterpret_cast<uintptr_t>(src) % 16 || !sink)
        return -1;
    hipLaunchKernelGGL(hbm_probe_read16, dim3(blocks), dim3(256), 0,
                       static_cast<hipStream_t>(stream), static_cast<const u32x4_t *>(src),
                       static_cast<unsigned *>(sink), bytes / 16);
    return hipGetLastError() == hipSuccess ? 0 : -2;
}
