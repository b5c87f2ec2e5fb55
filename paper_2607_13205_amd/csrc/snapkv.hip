// SnapKV windowed score with fused GQA sum and prefix max-pool: streaming
// two-pass kernels.
//
// Paper: §2 (SnapKV: windowed mass over the last W queries, 1-D max-pool over
// the KV axis), §4 "SnapKV mechanism" (pool kernel 7) and Algorithm 1
// (windowed-mass and pooling steps).
//
// A segment is one (layer, sample, KV head); its rows are the G*W window
// queries of the group (head-major), taken in row groups of 128 (a virtual
// segment, vseg, is one segment and one row group).  A workgroup of four waves
// owns a vseg and a contiguous range of its keys; each wave owns a 32-row
// block whose query fragments stay in registers.  Keys stream through a
// four-slot LDS ring in chunks of 64 with direct-to-LDS loads issued three
// chunks ahead, so every wave keeps HBM requests in flight while it multiplies
// on the matrix cores (bf16 32x32x16, fp32 32x32x2).  No workgroup waits on
// another one.
//
//   pass 1   snap_pass1    S^T = K Q^T: each lane holds one row and 16 keys per
//                          block, so the running row max and sum of
//                          exp2(x - max) stay in the lane; one log-sum-exp
//                          per (vseg, range, row) is written.
//   combine  snap_combine  per row: lse2 over the ranges (+inf for padding rows).
//   pass 2   snap_pass2    S = Q K^T: each lane holds one key and 16 rows, so
//                          the column sum of exp2(x - lse2) is a lane sum plus
//                          one shuffle; the four row blocks add through LDS.
//   pool     snap_pool     adds the row groups and max-pools the prefix.
//
// Logits are kept in log2 units (x = scale * log2(e) * <q, k>) so that every
// exponential is a single v_exp_f32.
#include "kve_device.h"
#include "kve_internal.h"
#include "kve_stream.h"

namespace kve {
namespace {

constexpr int kThreads = 256;  // four waves
constexpr int kWaves = 4;
constexpr int kRing = 4;       // LDS chunk slots: the chunk in use and three ahead
constexpr int kPoolTile = 256;
constexpr int kMaxPoolHalf = 127;

// Wait until this wave's loads of the current chunk have landed, while the
// loads of up to `ahead` later chunks stay in flight.
template <int LPW>
__device__ __forceinline__ void wait_chunk(int ahead) {
    if (ahead >= 2)
        wait_vmcnt<2 * LPW>();
    else if (ahead == 1)
        wait_vmcnt<LPW>();
    else
        wait_vmcnt<0>();
}

struct Span {
    int vseg, seg, rg, range, t_begin, t_end, nsub;
};

__device__ __forceinline__ Span span_of(int nranges, int rgroups, int range_keys, int N) {
    Span s;
    s.vseg = blockIdx.x / nranges;
    s.range = blockIdx.x - s.vseg * nranges;
    s.seg = s.vseg / rgroups;
    s.rg = s.vseg - s.seg * rgroups;
    s.t_begin = s.range * range_keys;
    s.t_end = min(N, s.t_begin + range_keys);
    s.nsub = (s.t_end - s.t_begin + kChunkKeys - 1) / kChunkKeys;
    return s;
}

template <typename T, int D>
__device__ __forceinline__ void load_q(QFrag<T, D>& qf, const T* q, int seg, int rows, int row) {
    using M = Mma<T>;
    const int lane = threadIdx.x & 63;
    const T* base = q + ((size_t)seg * rows + row) * D;
#pragma unroll
    for (int s = 0; s < KChunk<T, D>::NSTEP; ++s)
        qf[s] = row < rows ? M::load(base, s * M::KSTEP + (lane >> 5) * M::KPL) : M::zero();
}

template <typename T, int D>
__device__ __forceinline__ void issue_chunk(char* ring, const char* kseg, const Span& sp, int s) {
    const int t0 = sp.t_begin + s * kChunkKeys;
    chunk_stream<T, D, kWaves>(ring + (s % kRing) * KChunk<T, D>::BYTES, kseg + (size_t)t0 * KChunk<T, D>::ROW,
                               sp.t_end - t0, threadIdx.x >> 6, threadIdx.x & 63);
}

template <typename T, int D>
__global__ __launch_bounds__(kThreads, 2) void snap_pass1(const T* __restrict__ q, const T* __restrict__ k,
                                                          int N, int W, int rows, int rgroups, int nranges,
                                                          int range_keys, float sl2,
                                                          float* __restrict__ stats) {
    using C = KChunk<T, D>;
    using M = Mma<T>;
    constexpr int LPW = chunk_loads_per_wave<T, D, kWaves>();
    __shared__ __align__(16) char ring[kRing][C::BYTES];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const Span sp = span_of(nranges, rgroups, range_keys, N);
    const int P_rows = N - W;
    const char* kseg = reinterpret_cast<const char*>(k) + (size_t)sp.seg * N * C::ROW;

    QFrag<T, D> qf;
    const int qr = sp.rg * 128 + wave * 32 + (lane & 31);  // this lane's query row
    load_q<T, D>(qf, q, sp.seg, rows, qr);
    const int lim = qr < rows ? P_rows + (qr % W) : -1;
    drain_loads();

    for (int s = 0; s < min(kRing - 1, sp.nsub); ++s) issue_chunk<T, D>(&ring[0][0], kseg, sp, s);

    float m2 = -INFINITY, l = 0.0f;  // running max (log2 units) and sum of this lane's keys
    for (int s = 0; s < sp.nsub; ++s) {
        wait_chunk<LPW>(min(kRing - 2, sp.nsub - 1 - s));
        lds_barrier();
        if (s + kRing - 1 < sp.nsub) issue_chunk<T, D>(&ring[0][0], kseg, sp, s + kRing - 1);
        const char* buf = ring[s % kRing];
        const int t0 = sp.t_begin + s * kChunkKeys;
        float x[2][16];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            f32x16 acc = {};
            const int r = 32 * j + (lane & 31);
#pragma unroll
            for (int st = 0; st < C::NSTEP; ++st)
                acc = M::mma(chunk_frag<T, D>(buf, r, st * M::KSTEP + (lane >> 5) * M::KPL), qf[st], acc);
#pragma unroll
            for (int i = 0; i < 16; ++i) x[j][i] = acc[i];
        }
        if (t0 + kChunkKeys > P_rows) {  // keys past N or inside the causal window
#pragma unroll
            for (int j = 0; j < 2; ++j)
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int t = t0 + 32 * j + c_row(i, lane);
                    if (!(t < sp.t_end && t <= lim)) x[j][i] = -INFINITY;
                }
        }
        float mx = -INFINITY;
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int i = 0; i < 16; i += 2) mx = fmaxf(mx, fmaxf(x[j][i], x[j][i + 1]));
        const float mn = fmaxf(m2, mx * sl2);
        if (mn != -INFINITY) {
            float acc = l * fast_exp2(m2 - mn);
#pragma unroll
            for (int j = 0; j < 2; ++j)
#pragma unroll
                for (int i = 0; i < 16; ++i) acc += fast_exp2(fmaf(x[j][i], sl2, -mn));
            l = acc;
            m2 = mn;
        }
    }
    // the two lane halves hold the same row and different keys
    lse2_merge(m2, l, __shfl_xor(m2, 32), __shfl_xor(l, 32));
    if (lane < 32)
        stats[((size_t)sp.vseg * nranges + sp.range) * 128 + wave * 32 + lane] =
            (m2 != -INFINITY && l > 0.0f) ? m2 + log2f(l) : -INFINITY;
}

__global__ __launch_bounds__(128) void snap_combine(const float* __restrict__ stats, int nranges, int rows,
                                                    int rgroups, float* __restrict__ lse) {
    const int vseg = blockIdx.x, r = threadIdx.x;
    const int row = (vseg % rgroups) * 128 + r;
    float a = -INFINITY, b = 0.0f;
    for (int c = 0; c < nranges; ++c) {
        const float v = stats[((size_t)vseg * nranges + c) * 128 + r];
        lse2_merge(a, b, v, v == -INFINITY ? 0.0f : 1.0f);
    }
    // rows past the window rows contribute nothing to the column sums
    lse[(size_t)vseg * 128 + r] = (row < rows && b > 0.0f) ? a + log2f(b) : INFINITY;
}

template <typename T, int D>
__global__ __launch_bounds__(kThreads, 2) void snap_pass2(const T* __restrict__ q, const T* __restrict__ k,
                                                          int N, int W, int rows, int rgroups, int nranges,
                                                          int range_keys, float sl2,
                                                          const float* __restrict__ lse, int segs,
                                                          float* __restrict__ raw) {
    using C = KChunk<T, D>;
    using M = Mma<T>;
    constexpr int LPW = chunk_loads_per_wave<T, D, kWaves>();
    __shared__ __align__(16) char ring[kRing][C::BYTES];
    __shared__ float scol[2][kWaves][kChunkKeys];
    __shared__ float sraw[kSnapMaxRange];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const Span sp = span_of(nranges, rgroups, range_keys, N);
    const int P_rows = N - W;
    const char* kseg = reinterpret_cast<const char*>(k) + (size_t)sp.seg * N * C::ROW;

    QFrag<T, D> qf;
    const int row0 = sp.rg * 128 + wave * 32;
    load_q<T, D>(qf, q, sp.seg, rows, row0 + (lane & 31));
    float l2[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) l2[i] = lse[(size_t)sp.vseg * 128 + wave * 32 + c_row(i, lane)];
    drain_loads();

    for (int s = 0; s < min(kRing - 1, sp.nsub); ++s) issue_chunk<T, D>(&ring[0][0], kseg, sp, s);

    for (int s = 0; s < sp.nsub; ++s) {
        wait_chunk<LPW>(min(kRing - 2, sp.nsub - 1 - s));
        lds_barrier();
        if (s + kRing - 1 < sp.nsub) issue_chunk<T, D>(&ring[0][0], kseg, sp, s + kRing - 1);
        if (s >= 1 && tid < kChunkKeys) {
            const float* c = &scol[(s - 1) & 1][0][tid];
            sraw[(s - 1) * kChunkKeys + tid] =
                (c[0] + c[kChunkKeys]) + (c[2 * kChunkKeys] + c[3 * kChunkKeys]);
        }
        const char* buf = ring[s % kRing];
        const int t0 = sp.t_begin + s * kChunkKeys;
        const bool full = t0 + kChunkKeys <= P_rows;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            f32x16 acc = {};
            const int r = 32 * j + (lane & 31);
#pragma unroll
            for (int st = 0; st < C::NSTEP; ++st)
                acc = M::mma(qf[st], chunk_frag<T, D>(buf, r, st * M::KSTEP + (lane >> 5) * M::KPL), acc);
            float col = 0.0f;
            if (full) {
#pragma unroll
                for (int i = 0; i < 16; ++i) col += fast_exp2(fmaf(acc[i], sl2, -l2[i]));
            } else {
                const int t = t0 + r;
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int row = row0 + c_row(i, lane);
                    const bool ok = t < sp.t_end && row < rows && t <= P_rows + (row % W);
                    col += ok ? fast_exp2(fmaf(acc[i], sl2, -l2[i])) : 0.0f;
                }
            }
            col += __shfl_xor(col, 32);
            if (lane < 32) scol[s & 1][wave][32 * j + lane] = col;
        }
    }
    __syncthreads();
    if (tid < kChunkKeys) {
        const int s = sp.nsub - 1;
        const float* c = &scol[s & 1][0][tid];
        sraw[s * kChunkKeys + tid] = (c[0] + c[kChunkKeys]) + (c[2 * kChunkKeys] + c[3 * kChunkKeys]);
    }
    __syncthreads();
    float* out = raw + ((size_t)sp.rg * segs + sp.seg) * N + sp.t_begin;
    for (int e = tid; e < sp.t_end - sp.t_begin; e += kThreads) out[e] = sraw[e];
}

__global__ __launch_bounds__(kPoolTile) void snap_pool(const float* __restrict__ raw, int rgroups,
                                                       int segs, int N, int W, int pool_k, int tiles,
                                                       float* __restrict__ score) {
    __shared__ float ss[kPoolTile + 2 * kMaxPoolHalf];
    const int tile = blockIdx.x % tiles;
    const int seg = blockIdx.x / tiles;
    const int h = pool_k / 2;
    const int P = N - W;
    const int t0 = tile * kPoolTile;
    for (int e = threadIdx.x; e < kPoolTile + 2 * h; e += kPoolTile) {
        const int u = t0 - h + e;
        float s = -INFINITY;
        if (u >= 0 && u < N) {
            s = 0.0f;
            for (int rg = 0; rg < rgroups; ++rg) s += raw[((size_t)rg * segs + seg) * N + u];
        }
        ss[e] = s;
    }
    __syncthreads();
    const int t = t0 + threadIdx.x;
    if (t >= N) return;
    float v;
    if (t < P) {
        const int lo = max(0, t - h), hi = min(P - 1, t + h);
        v = -INFINITY;
        for (int u = lo; u <= hi; ++u) v = fmaxf(v, ss[u - t0 + h]);
    } else {
        v = ss[threadIdx.x + h];
    }
    score[(size_t)seg * N + t] = v;
}

template <typename T, int D>
hipError_t run_snapkv(const void* q, const void* k, int L, int B, int Hq, int Hkv, int N, int W,
                      float scale, int pool_k, float* score, void* ws, bool persistent, hipStream_t st) {
    const SnapPlan p = snap_plan(L, B, Hq, Hkv, N, W, D);
    char* w = static_cast<char*>(ws);
    float* stats = reinterpret_cast<float*>(w + p.off_stats);
    float* lse = reinterpret_cast<float*>(w + p.off_lse);
    float* raw = reinterpret_cast<float*>(w + p.off_raw);
    const float sl2 = scale * kLog2e;
    const T* qt = static_cast<const T*>(q);
    const T* kt = static_cast<const T*>(k);
    bool used = false;
    if (persistent) {
        const hipError_t e = launch_snapkv_fused(q, k, sizeof(T) == 2 ? 0 : 1, L, B, Hq, Hkv, N, W, D, scale,
                                                 raw, ws, st, &used);
        if (e != hipSuccess) return e;
    }
    if (!used) {
        const dim3 grid((unsigned)((size_t)p.n_vsegs * p.nranges));
        hipLaunchKernelGGL((snap_pass1<T, D>), grid, dim3(kThreads), 0, st, qt, kt, N, W, p.rows, p.rgroups,
                           p.nranges, p.range_keys, sl2, stats);
        hipLaunchKernelGGL(snap_combine, dim3((unsigned)p.n_vsegs), dim3(128), 0, st, stats, p.nranges, p.rows,
                           p.rgroups, lse);
        hipLaunchKernelGGL((snap_pass2<T, D>), grid, dim3(kThreads), 0, st, qt, kt, N, W, p.rows, p.rgroups,
                           p.nranges, p.range_keys, sl2, lse, p.segs, raw);
    }
    const int tiles = (N + kPoolTile - 1) / kPoolTile;
    hipLaunchKernelGGL(snap_pool, dim3((unsigned)(p.segs * tiles)), dim3(kPoolTile), 0, st, raw,
                       p.rgroups, p.segs, N, W, pool_k, tiles, score);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_snapkv(const void* q, const void* k, int dtype, int L, int B, int Hq, int Hkv,
                         int N, int W, int d, float scale, int pool_k, float* score, void* ws,
                         bool persistent, hipStream_t st) {
    if (dtype == 0) {
        if (d == 128)
            return run_snapkv<__bf16, 128>(q, k, L, B, Hq, Hkv, N, W, scale, pool_k, score, ws, persistent, st);
        return run_snapkv<__bf16, 64>(q, k, L, B, Hq, Hkv, N, W, scale, pool_k, score, ws, persistent, st);
    }
    if (d == 128)
        return run_snapkv<float, 128>(q, k, L, B, Hq, Hkv, N, W, scale, pool_k, score, ws, persistent, st);
    return run_snapkv<float, 64>(q, k, L, B, Hq, Hkv, N, W, scale, pool_k, score, ws, persistent, st);
}

}  // namespace kve
