// Streaming copy, read and fill kernels of known traffic, used by the
// benchmark as the measured HBM ceilings of this GPU (read only; read +
// write; write only) and as the reference kernel that scales the rocprofv3
// FETCH_SIZE / WRITE_SIZE counters to bytes.  Not part of the routing ABI.
//
// Each lane keeps U independent 16-byte loads in flight: a workgroup covers
// 256 U consecutive vectors per step (U coalesced 4 KB rows), then strides
// over the grid.  Loads and stores are non-temporal (streaming).
#include <hip/hip_runtime.h>

typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));

template <int U>
__global__ void __launch_bounds__(256)
hbm_probe_copy16(const u32x4_t *__restrict__ src, u32x4_t *__restrict__ dst, long long n)
{
    const long long stride = (long long)gridDim.x * 256 * U;
    for (long long base = (long long)blockIdx.x * 256 * U + threadIdx.x; base < n;
         base += stride) {
        u32x4_t v[U];
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (base + u * 256 < n)
                v[u] = __builtin_nontemporal_load(src + base + u * 256);
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (base + u * 256 < n)
                __builtin_nontemporal_store(v[u], dst + base + u * 256);
    }
}

template <int U>
__global__ void __launch_bounds__(256)
hbm_probe_read16(const u32x4_t *__restrict__ src, unsigned *__restrict__ sink, long long n)
{
    const long long stride = (long long)gridDim.x * 256 * U;
    unsigned acc = 0;
    for (long long base = (long long)blockIdx.x * 256 * U + threadIdx.x; base < n;
         base += stride) {
        u32x4_t v[U];
#pragma unroll
        for (int u = 0; u < U; ++u)
            v[u] = base + u * 256 < n ? __builtin_nontemporal_load(src + base + u * 256)
                                      : u32x4_t{0u, 0u, 0u, 0u};
#pragma unroll
        for (int u = 0; u < U; ++u)
            acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
    if (acc == 0x9e3779b9u)  // keeps the loads; practically never true
        sink[0] = acc;
}

template <int U>
__global__ void __launch_bounds__(256)
hbm_probe_fill16(u32x4_t *__restrict__ dst, long long n)
{
    const long long stride = (long long)gridDim.x * 256 * U;
    const u32x4_t v = {1u, 2u, 3u, 4u};
    for (long long base = (long long)blockIdx.x * 256 * U + threadIdx.x; base < n;
         base += stride)
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (base + u * 256 < n)
                dst[base + u * 256] = v;
}

namespace {

bool bad_args(const void *a, const void *b, long long bytes, int blocks)
{
    return bytes % 16 || bytes < 0 || blocks < 1 ||
           (reinterpret_cast<uintptr_t>(a) | reinterpret_cast<uintptr_t>(b)) % 16;
}

}  // namespace

// bytes must be a multiple of 16 and the pointers 16-byte aligned; unroll
// is the number of loads in flight per lane (1, 2, 4 or 8).  0 on success.
extern "C" int hbm_probe_copy_u(const void *src, void *dst, long long bytes, int blocks,
                                int unroll, void *stream)
{
    if (bad_args(src, dst, bytes, blocks) || !src || !dst)
        return -1;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const u32x4_t *a = static_cast<const u32x4_t *>(src);
    u32x4_t *b = static_cast<u32x4_t *>(dst);
    const long long n = bytes / 16;
    switch (unroll) {
    case 1: hipLaunchKernelGGL(hbm_probe_copy16<1>, dim3(blocks), dim3(256), 0, st, a, b, n); break;
    case 2: hipLaunchKernelGGL(hbm_probe_copy16<2>, dim3(blocks), dim3(256), 0, st, a, b, n); break;
    case 4: hipLaunchKernelGGL(hbm_probe_copy16<4>, dim3(blocks), dim3(256), 0, st, a, b, n); break;
    case 8: hipLaunchKernelGGL(hbm_probe_copy16<8>, dim3(blocks), dim3(256), 0, st, a, b, n); break;
    default: return -1;
    }
    return hipGetLastError() == hipSuccess ? 0 : -2;
}

extern "C" int hbm_probe_read_u(const void *src, void *sink, long long bytes, int blocks,
                                int unroll, void *stream)
{
    if (bad_args(src, sink, bytes, blocks) || !src || !sink)
        return -1;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const u32x4_t *a = static_cast<const u32x4_t *>(src);
    unsigned *s = static_cast<unsigned *>(sink);
    const long long n = bytes / 16;
    switch (unroll) {
    case 1: hipLaunchKernelGGL(hbm_probe_read16<1>, dim3(blocks), dim3(256), 0, st, a, s, n); break;
    case 2: hipLaunchKernelGGL(hbm_probe_read16<2>, dim3(blocks), dim3(256), 0, st, a, s, n); break;
    case 4: hipLaunchKernelGGL(hbm_probe_read16<4>, dim3(blocks), dim3(256), 0, st, a, s, n); break;
    case 8: hipLaunchKernelGGL(hbm_probe_read16<8>, dim3(blocks), dim3(256), 0, st, a, s, n); break;
    default: return -1;
    }
    return hipGetLastError() == hipSuccess ? 0 : -2;
}

extern "C" int hbm_probe_fill_u(void *dst, long long bytes, int blocks, int unroll, void *stream)
{
    if (bad_args(dst, dst, bytes, blocks) || !dst)
        return -1;
    hipStream_t st = static_cast<hipStream_t>(stream);
    u32x4_t *b = static_cast<u32x4_t *>(dst);
    const long long n = bytes / 16;
    switch (unroll) {
    case 1: hipLaunchKernelGGL(hbm_probe_fill16<1>, dim3(blocks), dim3(256), 0, st, b, n); break;
    case 4: hipLaunchKernelGGL(hbm_probe_fill16<4>, dim3(blocks), dim3(256), 0, st, b, n); break;
    default: return -1;
    }
    return hipGetLastError() == hipSuccess ? 0 : -2;
}

// The reference copy of the counter runs: one load per lane in flight.
extern "C" int hbm_probe_copy(const void *src, void *dst, long long bytes, int blocks,
                              void *stream)
{
    return hbm_probe_copy_u(src, dst, bytes, blocks, 1, stream);
}

extern "C" int hbm_probe_read(const void *src, void *sink, long long bytes, int blocks,
                              void *stream)
{
    return hbm_probe_read_u(src, sink, bytes, blocks, 8, stream);
}
