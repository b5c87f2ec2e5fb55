// Read-bandwidth probe: the measurement helper the benchmark times next to the
// eviction kernels (not part of the eviction path).  Every byte of a buffer is
// read once with 16-byte loads, eight in flight per thread, by a fixed grid
// that strides over the buffer; each workgroup writes one value derived from
// what it read, so that no load can be dropped.  Over a buffer far larger than
// the last-level cache it gives the streaming HBM read rate; repeated over a
// buffer that fits in that cache (but not in the L2s), the cache's re-read rate.
#include "kve_device.h"
#include "kve_internal.h"

namespace kve {
namespace {

constexpr int kProbeThreads = 256;
constexpr int kProbeUnroll = 8;

template <bool NT>
__global__ __launch_bounds__(kProbeThreads) void read_probe(const u32x4* __restrict__ buf, size_t n16,
                                                            float* __restrict__ sink) {
    const size_t stride = (size_t)gridDim.x * kProbeThreads;
    size_t i = (size_t)blockIdx.x * kProbeThreads + threadIdx.x;
    uint32_t acc = 0u;
    for (; i + (kProbeUnroll - 1) * stride < n16; i += kProbeUnroll * stride) {
        u32x4 v[kProbeUnroll];
#pragma unroll
        for (int u = 0; u < kProbeUnroll; ++u)
            v[u] = NT ? __builtin_nontemporal_load(buf + i + u * stride) : buf[i + u * stride];
#pragma unroll
        for (int u = 0; u < kProbeUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
    for (; i < n16; i += stride) {
        const u32x4 v = buf[i];
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    // one value per workgroup (the xor of its lanes' words, as a float's bits)
    for (int o = 32; o > 0; o >>= 1) acc ^= (uint32_t)__shfl_xor((int)acc, o);
    __shared__ uint32_t part[kProbeThreads / 64];
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t a = 0u;
        for (int w = 0; w < kProbeThreads / 64; ++w) a ^= part[w];
        sink[blockIdx.x] = __uint_as_float(a & 0x007fffffu);  // a finite float
    }
}

}  // namespace

hipError_t launch_read_probe(const void* buf, size_t bytes, int nontemporal, float* sink, int blocks,
                             hipStream_t st) {
    const size_t n16 = bytes / 16;
    const auto* b = static_cast<const u32x4*>(buf);
    if (nontemporal)
        hipLaunchKernelGGL(read_probe<true>, dim3((unsigned)blocks), dim3(kProbeThreads), 0, st, b, n16, sink);
    else
        hipLaunchKernelGGL(read_probe<false>, dim3((unsigned)blocks), dim3(kProbeThreads), 0, st, b, n16, sink);
    return hipGetLastError();
}

}  // namespace kve
