// Linear role probe (§6 "Deployment: a linear role probe"): the role label of
// every token from a multinomial logistic regression over the token ids at
// t-2 .. t+2.  One thread per token: five gathers of an R-float row from the
// weight tables (a few MB, resident in L2 and the last-level cache after the
// first touch), a float32 sum in a fixed order and an argmax.
#include "kve_device.h"
#include "kve_internal.h"

namespace kve {
namespace {

constexpr int kThreads = 256;
constexpr int kOffsets = 5;  // t-2 .. t+2

template <int R>
__global__ __launch_bounds__(kThreads) void probe_kernel(const int32_t* __restrict__ ids, int N, long long total,
                                                         const float* __restrict__ weight,
                                                         const float* __restrict__ bias, int V,
                                                         int8_t* __restrict__ out) {
    const long long i = (long long)blockIdx.x * kThreads + threadIdx.x;
    if (i >= total) return;
    const long long row = i / N;
    const int pos = (int)(i - row * N);
    const int32_t* seq = ids + row * N;
    float acc[R];
#pragma unroll
    for (int r = 0; r < R; ++r) acc[r] = bias[r];
    // bias first, then the offsets in order: the same float32 sum everywhere
#pragma unroll
    for (int o = 0; o < kOffsets; ++o) {
        const int p = pos + o - 2;
        if (p < 0 || p >= N) continue;
        const int id = seq[p];
        if (id < 0 || id >= V) continue;
        const float* w = weight + ((size_t)o * V + id) * R;
#pragma unroll
        for (int r = 0; r < R; ++r) acc[r] = __fadd_rn(acc[r], w[r]);
    }
    int best = 0;
#pragma unroll
    for (int r = 1; r < R; ++r)
        if (acc[r] > acc[best]) best = r;  // the first maximum wins ties
    out[i] = (int8_t)best;
}

template <int R>
hipError_t run_probe(const int32_t* ids, int B, int N, const float* weight, const float* bias, int V,
                     int8_t* out, hipStream_t st) {
    const long long total = (long long)B * N;
    hipLaunchKernelGGL((probe_kernel<R>), dim3((unsigned)((total + kThreads - 1) / kThreads)), dim3(kThreads), 0,
                       st, ids, N, total, weight, bias, V, out);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_probe(const int32_t* ids, int B, int N, const float* weight, const float* bias, int V, int R,
                        int8_t* out, hipStream_t st) {
    switch (R) {
        case 1: return run_probe<1>(ids, B, N, weight, bias, V, out, st);
        case 2: return run_probe<2>(ids, B, N, weight, bias, V, out, st);
        case 3: return run_probe<3>(ids, B, N, weight, bias, V, out, st);
        case 4: return run_probe<4>(ids, B, N, weight, bias, V, out, st);
        case 5: return run_probe<5>(ids, B, N, weight, bias, V, out, st);
        case 6: return run_probe<6>(ids, B, N, weight, bias, V, out, st);
        case 7: return run_probe<7>(ids, B, N, weight, bias, V, out, st);
        default: return run_probe<8>(ids, B, N, weight, bias, V, out, st);
    }
}

}  // namespace kve
