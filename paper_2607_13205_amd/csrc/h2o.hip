// H2O accumulated attention score, the baseline scorer.
//
// Paper §2 (H2O family): s(t) = sum over prefill queries q of p_t(q), kept per
// (layer, head); here summed over the G query heads of each KV head.
//
// The causal QK^T is a dense contraction, so both passes run on the matrix
// cores (bf16 32x32x16, fp32 32x32x2):
//   h2o_rows  one workgroup per (query head, 128-row block): four waves own 32
//             rows each (query fragments in registers) and stream the causal
//             keys through LDS; per row m + log2(sum exp2(x - m)).
//   h2o_cols  one workgroup per (KV head, 128-key block): four waves own 32 keys
//             each (key fragments in registers) and stream every later query
//             row of the G heads, with its log-sum-exp, through LDS; per key
//             sum of exp2(x - lse2).
// Logits are in log2 units, x = scale * log2(e) * <q, k>.
#include "kve_device.h"
#include "kve_internal.h"

namespace kve {
namespace {

constexpr int kThreads = 256;
constexpr int kTile = 64;  // keys (rows pass) or query rows (cols pass) per LDS tile

template <typename T, int D>
struct H2oShape {
    static constexpr int ES = (int)sizeof(T);
    static constexpr int ROW_BYTES = D * ES;
    static constexpr int ROWB = ROW_BYTES + 16;
    static constexpr int TILE_BYTES = kTile * ROW_BYTES;
    static constexpr int NSTEP = D / Mma<T>::KSTEP;
};

template <typename T, int D>
using FragArr = typename Mma<T>::frag[H2oShape<T, D>::NSTEP];


template <typename T, int D>
__device__ __forceinline__ void stage_tile(char* dst, const T* src, int t0, int t_end) {
    using S = H2oShape<T, D>;
    for (int o = threadIdx.x * 16; o < S::TILE_BYTES; o += kThreads * 16) {
        const int row = o / S::ROW_BYTES;
        const int within = o - row * S::ROW_BYTES;
        const int t = t0 + row;
        u32x4 v = zero16();
        if (t < t_end)
            v = ld16(reinterpret_cast<const char*>(src) + (size_t)t * S::ROW_BYTES + within);
        st16(dst + row * S::ROWB + within, v);
    }
}

template <typename T, int D>
__device__ __forceinline__ void load_frags(FragArr<T, D>& fr,
                                           const T* base, int row, int nrows) {
    using M = Mma<T>;
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int s = 0; s < H2oShape<T, D>::NSTEP; ++s) {
        const int kb = s * M::KSTEP + (lane >> 5) * M::KPL;
        fr[s] = row < nrows ? M::load(base + (size_t)row * D, kb) : M::zero();
    }
}

template <typename T, int D>
__global__ __launch_bounds__(kThreads) void h2o_rows(const T* __restrict__ q, const T* __restrict__ k,
                                                     int Hq, int Hkv, int N, int nrb, float sl2,
                                                     float* __restrict__ lse) {
    using S = H2oShape<T, D>;
    using M = Mma<T>;
    __shared__ __align__(16) char sk[kTile * S::ROWB];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int bid = blockIdx.x;
    const int rb = nrb - 1 - bid % nrb;  // longest causal rows first
    bid /= nrb;
    const int hq = bid % Hq;
    const int lb = bid / Hq;
    const int G = Hq / Hkv;
    const int j = hq / G;
    const int row0 = rb * kH2oRowBlock + wave * 32;
    const T* qh = q + ((size_t)lb * Hq + hq) * N * D;
    const T* kj = k + ((size_t)lb * Hkv + j) * N * D;

    typename M::frag qa[S::NSTEP];
    load_frags<T, D>(qa, qh, row0 + (lane & 31), N);
    float m[16], l[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        m[i] = -INFINITY;
        l[i] = 0.0f;
    }
    const int t_end = min(N, rb * kH2oRowBlock + kH2oRowBlock);
    for (int t0 = 0; t0 < t_end; t0 += kTile) {
        __syncthreads();
        stage_tile<T, D>(sk, kj, t0, t_end);
        __syncthreads();
        if (row0 >= N) continue;
#pragma unroll
        for (int cb = 0; cb < kTile / 32; ++cb) {
            if (t0 + cb * 32 > row0 + 31) continue;  // every key of the block is after every row
            f32x16 acc = {};
            const char* krow = sk + (cb * 32 + (lane & 31)) * S::ROWB;
#pragma unroll
            for (int s = 0; s < S::NSTEP; ++s)
                acc = M::mma(qa[s], M::load(krow, s * M::KSTEP + (lane >> 5) * M::KPL), acc);
            const int t = t0 + cb * 32 + (lane & 31);
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int r = row0 + c_row(i, lane);
                const bool valid = r < N && t <= r;
                const float x = valid ? acc[i] * sl2 : -INFINITY;
                const float mn = fmaxf(m[i], x);
                if (mn != -INFINITY) {
                    l[i] = l[i] * fast_exp2(m[i] - mn) + fast_exp2(x - mn);
                    m[i] = mn;
                }
            }
        }
    }
#pragma unroll
    for (int off = 1; off < 32; off <<= 1) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const float mo = __shfl_xor(m[i], off);
            const float lo = __shfl_xor(l[i], off);
            lse2_merge(m[i], l[i], mo, lo);
        }
    }
    if ((lane & 31) == 0) {
        float* out = lse + ((size_t)lb * Hq + hq) * N;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int r = row0 + c_row(i, lane);
            if (r < N) out[r] = l[i] > 0.0f ? m[i] + log2f(l[i]) : -INFINITY;
        }
    }
}

template <typename T, int D>
__global__ __launch_bounds__(kThreads) void h2o_cols(const T* __restrict__ q, const T* __restrict__ k,
                                                     const float* __restrict__ lse, int Hq, int Hkv,
                                                     int N, int nkb, float sl2,
                                                     float* __restrict__ score) {
    using S = H2oShape<T, D>;
    using M = Mma<T>;
    __shared__ __align__(16) char sq[kTile * S::ROWB];
    __shared__ float slse[kTile];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int bid = blockIdx.x;
    const int kb = bid % nkb;
    bid /= nkb;
    const int j = bid % Hkv;
    const int lb = bid / Hkv;
    const int G = Hq / Hkv;
    const int key0 = kb * kH2oKeyBlock + wave * 32;
    const int my_key = key0 + (lane & 31);
    const T* kj = k + ((size_t)lb * Hkv + j) * N * D;

    typename M::frag kf[S::NSTEP];
    load_frags<T, D>(kf, kj, my_key, N);
    float col = 0.0f;
    const int r_start = (kb * kH2oKeyBlock) / kTile * kTile;
    for (int h = 0; h < G; ++h) {
        const size_t head = (size_t)lb * Hq + (size_t)j * G + h;
        const T* qh = q + head * N * D;
        const float* lh = lse + head * N;
        for (int r0 = r_start; r0 < N; r0 += kTile) {
            __syncthreads();
            stage_tile<T, D>(sq, qh, r0, N);
            if (threadIdx.x < kTile) {
                const int r = r0 + threadIdx.x;
                slse[threadIdx.x] = r < N ? lh[r] : 0.0f;
            }
            __syncthreads();
            if (key0 >= N || r0 + kTile - 1 < key0) continue;
#pragma unroll
            for (int rbk = 0; rbk < kTile / 32; ++rbk) {
                if (r0 + rbk * 32 + 31 < key0) continue;  // every row of the block is before every key
                f32x16 acc = {};
                const char* qrow = sq + (rbk * 32 + (lane & 31)) * S::ROWB;
#pragma unroll
                for (int s = 0; s < S::NSTEP; ++s)
                    acc = M::mma(M::load(qrow, s * M::KSTEP + (lane >> 5) * M::KPL), kf[s], acc);
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int rr = rbk * 32 + c_row(i, lane);
                    const int r = r0 + rr;
                    const bool valid = r < N && r >= my_key;
                    col += valid ? fast_exp2(acc[i] * sl2 - slse[rr]) : 0.0f;
                }
            }
        }
    }
    col += __shfl_xor(col, 32);
    if (lane < 32 && my_key < N) score[((size_t)lb * Hkv + j) * N + my_key] = col;
}

template <typename T, int D>
hipError_t run_h2o(const void* q, const void* k, int L, int B, int Hq, int Hkv, int N, float scale,
                   float* score, void* ws, hipStream_t st) {
    float* lse = static_cast<float*>(ws);
    const float sl2 = scale * kLog2e;
    const T* qt = static_cast<const T*>(q);
    const T* kt = static_cast<const T*>(k);
    const int nrb = (N + kH2oRowBlock - 1) / kH2oRowBlock;
    const int nkb = (N + kH2oKeyBlock - 1) / kH2oKeyBlock;
    hipLaunchKernelGGL((h2o_rows<T, D>), dim3((unsigned)((size_t)L * B * Hq * nrb)), dim3(kThreads), 0,
                       st, qt, kt, Hq, Hkv, N, nrb, sl2, lse);
    hipLaunchKernelGGL((h2o_cols<T, D>), dim3((unsigned)((size_t)L * B * Hkv * nkb)), dim3(kThreads), 0,
                       st, qt, kt, lse, Hq, Hkv, N, nkb, sl2, score);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_h2o(const void* q, const void* k, int dtype, int L, int B, int Hq, int Hkv, int N,
                      int d, float scale, float* score, void* ws, hipStream_t st) {
    if (dtype == 0) {
        if (d == 128) return run_h2o<__bf16, 128>(q, k, L, B, Hq, Hkv, N, scale, score, ws, st);
        return run_h2o<__bf16, 64>(q, k, L, B, Hq, Hkv, N, scale, score, ws, st);
    }
    if (d == 128) return run_h2o<float, 128>(q, k, L, B, Hq, Hkv, N, scale, score, ws, st);
    return run_h2o<float, 64>(q, k, L, B, Hq, Hkv, N, scale, score, ws, st);
}

}  // namespace kve
