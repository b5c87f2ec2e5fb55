// SnapKV windowed score with fused GQA sum and prefix max-pool.
//
// Paper: §2 (SnapKV: windowed mass over the last W queries, 1-D max-pool over
// the KV axis), §4 "SnapKV mechanism" (pool kernel 7) and Algorithm 1
// (windowed-mass and pooling steps).
//
// Work decomposition.  A segment is one (layer, sample, KV head).  Its rows are
// the G*W window queries of the group (head-major), taken in row groups of 128
// rows: one workgroup of four waves owns a row group and a chunk of keys; each
// wave owns a 32-row block whose query fragments stay in registers for the whole
// chunk.  Keys are streamed through LDS in tiles of 64 with 16-byte coalesced
// loads and multiplied on the matrix cores (bf16: 32x32x16, fp32: 32x32x2).
//
//   pass 1  snap_stats   per (chunk, row): running max m and sum of exp2(x - m)
//   combine snap_lse     per row: lse2 = m + log2(sum) over the chunks
//   pass 2  snap_colsum  per key: sum over the row group of exp2(x - lse2)
//   pool    snap_pool    adds the row groups and max-pools the prefix
//
// Logits are kept in log2 units (x = scale * log2(e) * <q, k>) so that every
// exponential is a single v_exp_f32.
#include "kve_device.h"
#include "kve_internal.h"

namespace kve {
namespace {

constexpr int kThreads = 256;
constexpr int kPoolTile = 256;
constexpr int kMaxPoolHalf = 127;

template <typename T, int D>
struct SnapShape {
    static constexpr int ES = (int)sizeof(T);
    static constexpr int ROW_BYTES = D * ES;
    static constexpr int ROWB = ROW_BYTES + 16;  // padded LDS row: spreads banks
    static constexpr int TILE_BYTES = kSnapTileKeys * ROW_BYTES;
    static constexpr int NSTEP = D / Mma<T>::KSTEP;
};

template <typename T, int D>
using FragArr = typename Mma<T>::frag[SnapShape<T, D>::NSTEP];


// Copy rows [t0, t0 + kSnapTileKeys) of a [*, D] matrix into LDS; rows at or
// beyond t_end are zero-filled.  All threads of the block take part.
template <typename T, int D>
__device__ __forceinline__ void stage_rows(char* dst, const T* src, int t0, int t_end) {
    using S = SnapShape<T, D>;
    for (int o = threadIdx.x * 16; o < S::TILE_BYTES; o += kThreads * 16) {
        const int key = o / S::ROW_BYTES;
        const int within = o - key * S::ROW_BYTES;
        const int t = t0 + key;
        u32x4 v = zero16();
        if (t < t_end)
            v = ld16(reinterpret_cast<const char*>(src) + (size_t)t * S::ROW_BYTES + within);
        st16(dst + key * S::ROWB + within, v);
    }
}

// Query fragments of this lane's row (A operand) for every k step.
template <typename T, int D>
__device__ __forceinline__ void load_row_frags(FragArr<T, D>& fr,
                                               const T* base, int row, int nrows) {
    using M = Mma<T>;
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int s = 0; s < SnapShape<T, D>::NSTEP; ++s) {
        const int kb = s * M::KSTEP + (lane >> 5) * M::KPL;
        fr[s] = row < nrows ? M::load(base + (size_t)row * D, kb) : M::zero();
    }
}

// 32 rows x 32 keys block: A fragments in registers, B rows in LDS.
template <typename T, int D>
__device__ __forceinline__ f32x16 block_logits(const FragArr<T, D>& qa,
                                               const char* krow) {
    using M = Mma<T>;
    const int lane = threadIdx.x & 63;
    f32x16 acc = {};
#pragma unroll
    for (int s = 0; s < SnapShape<T, D>::NSTEP; ++s)
        acc = M::mma(qa[s], M::load(krow, s * M::KSTEP + (lane >> 5) * M::KPL), acc);
    return acc;
}

struct SegIdx {
    int c, rg, seg;
};
__device__ __forceinline__ SegIdx seg_index(int nchunks, int rgroups) {
    int bid = blockIdx.x;
    SegIdx s;
    s.c = bid % nchunks;
    bid /= nchunks;
    s.rg = bid % rgroups;
    s.seg = bid / rgroups;
    return s;
}

template <typename T, int D>
__global__ __launch_bounds__(kThreads) void snap_stats(const T* __restrict__ q, const T* __restrict__ k,
                                                       int N, int W, int rows, int rgroups,
                                                       int rows_pad, int chunk, int nchunks, float sl2,
                                                       float2* __restrict__ stats) {
    using S = SnapShape<T, D>;
    __shared__ __align__(16) char sk[kSnapTileKeys * S::ROWB];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const SegIdx ix = seg_index(nchunks, rgroups);
    const int row0 = ix.rg * kSnapRowsPerGroup + wave * 32;
    const T* qseg = q + (size_t)ix.seg * rows * D;
    const T* kseg = k + (size_t)ix.seg * N * D;

    typename Mma<T>::frag qa[S::NSTEP];
    load_row_frags<T, D>(qa, qseg, row0 + (lane & 31), rows);

    float m[16], l[16];
    int lim[16];  // last key each of this lane's rows may see (causal), -1 for padding rows
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        const int r = row0 + c_row(i, lane);
        m[i] = -INFINITY;
        l[i] = 0.0f;
        lim[i] = r < rows ? N - W + (r % W) : -1;
    }
    const int t_begin = ix.c * chunk;
    const int t_end = min(N, t_begin + chunk);
    for (int t0 = t_begin; t0 < t_end; t0 += kSnapTileKeys) {
        __syncthreads();
        stage_rows<T, D>(sk, kseg, t0, t_end);
        __syncthreads();
        if (row0 >= rows) continue;
#pragma unroll
        for (int cb = 0; cb < kSnapTileKeys / 32; ++cb) {
            const f32x16 acc = block_logits<T, D>(qa, sk + (cb * 32 + (lane & 31)) * S::ROWB);
            const int t = t0 + cb * 32 + (lane & 31);
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const bool valid = t < t_end && t <= lim[i];
                const float x = valid ? acc[i] * sl2 : -INFINITY;
                const float mn = fmaxf(m[i], x);
                if (mn != -INFINITY) {
                    l[i] = l[i] * fast_exp2(m[i] - mn) + fast_exp2(x - mn);
                    m[i] = mn;
                }
            }
        }
    }
    // combine the 32 lanes that hold the same rows
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
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int r = row0 + c_row(i, lane);
            if (r < rows)
                stats[((size_t)ix.seg * nchunks + ix.c) * rows_pad + r] = make_float2(m[i], l[i]);
        }
    }
}

__global__ __launch_bounds__(kThreads) void snap_lse(const float2* __restrict__ stats, int nchunks,
                                                     int rows, int rows_pad, float* __restrict__ lse) {
    const int seg = blockIdx.x;
    for (int r = threadIdx.x; r < rows; r += blockDim.x) {
        float m = -INFINITY, l = 0.0f;
        for (int c = 0; c < nchunks; ++c) {
            const float2 v = stats[((size_t)seg * nchunks + c) * rows_pad + r];
            lse2_merge(m, l, v.x, v.y);
        }
        lse[(size_t)seg * rows_pad + r] = l > 0.0f ? m + log2f(l) : -INFINITY;
    }
}

template <typename T, int D>
__global__ __launch_bounds__(kThreads) void snap_colsum(const T* __restrict__ q, const T* __restrict__ k,
                                                        int N, int W, int rows, int rgroups,
                                                        int rows_pad, int chunk, int nchunks, float sl2,
                                                        const float* __restrict__ lse, int segs,
                                                        float* __restrict__ raw) {
    using S = SnapShape<T, D>;
    __shared__ __align__(16) char sk[kSnapTileKeys * S::ROWB];
    __shared__ float scol[kThreads / kWave][kSnapTileKeys];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const SegIdx ix = seg_index(nchunks, rgroups);
    const int row0 = ix.rg * kSnapRowsPerGroup + wave * 32;
    const T* qseg = q + (size_t)ix.seg * rows * D;
    const T* kseg = k + (size_t)ix.seg * N * D;

    typename Mma<T>::frag qa[S::NSTEP];
    load_row_frags<T, D>(qa, qseg, row0 + (lane & 31), rows);

    float lr[16];
    int lim[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        const int r = row0 + c_row(i, lane);
        lim[i] = r < rows ? N - W + (r % W) : -1;
        lr[i] = r < rows ? lse[(size_t)ix.seg * rows_pad + r] : 0.0f;
    }
    float* out = raw + ((size_t)ix.rg * segs + ix.seg) * N;
    const int t_begin = ix.c * chunk;
    const int t_end = min(N, t_begin + chunk);
    for (int t0 = t_begin; t0 < t_end; t0 += kSnapTileKeys) {
        __syncthreads();
        stage_rows<T, D>(sk, kseg, t0, t_end);
        __syncthreads();
        float col[kSnapTileKeys / 32];
#pragma unroll
        for (int cb = 0; cb < kSnapTileKeys / 32; ++cb) col[cb] = 0.0f;
        if (row0 < rows) {
#pragma unroll
            for (int cb = 0; cb < kSnapTileKeys / 32; ++cb) {
                const f32x16 acc = block_logits<T, D>(qa, sk + (cb * 32 + (lane & 31)) * S::ROWB);
                const int t = t0 + cb * 32 + (lane & 31);
                float sum = 0.0f;
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const bool valid = t < t_end && t <= lim[i];
                    sum += valid ? fast_exp2(acc[i] * sl2 - lr[i]) : 0.0f;
                }
                col[cb] = sum;
            }
        }
#pragma unroll
        for (int cb = 0; cb < kSnapTileKeys / 32; ++cb) {
            col[cb] += __shfl_xor(col[cb], 32);
            if (lane < 32) scol[wave][cb * 32 + lane] = col[cb];
        }
        __syncthreads();
        if (threadIdx.x < kSnapTileKeys) {
            const int t = t0 + threadIdx.x;
            if (t < t_end) {
                float s = 0.0f;
#pragma unroll
                for (int w = 0; w < kThreads / kWave; ++w) s += scol[w][threadIdx.x];
                out[t] = s;
            }
        }
    }
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
                      float scale, int pool_k, float* score, void* ws, hipStream_t st) {
    const SnapPlan p = snap_plan(L, B, Hq, Hkv, N, W);
    char* w = static_cast<char*>(ws);
    float2* stats = reinterpret_cast<float2*>(w + p.off_stats);
    float* lse = reinterpret_cast<float*>(w + p.off_lse);
    float* raw = reinterpret_cast<float*>(w + p.off_raw);
    const float sl2 = scale * kLog2e;
    const T* qt = static_cast<const T*>(q);
    const T* kt = static_cast<const T*>(k);
    const dim3 grid((unsigned)(p.segs * p.rgroups * p.nchunks));
    hipLaunchKernelGGL((snap_stats<T, D>), grid, dim3(kThreads), 0, st, qt, kt, N, W, p.rows,
                       p.rgroups, p.rows_pad, p.chunk, p.nchunks, sl2, stats);
    hipLaunchKernelGGL(snap_lse, dim3(p.segs), dim3(kThreads), 0, st, stats, p.nchunks, p.rows,
                       p.rows_pad, lse);
    hipLaunchKernelGGL((snap_colsum<T, D>), grid, dim3(kThreads), 0, st, qt, kt, N, W, p.rows,
                       p.rgroups, p.rows_pad, p.chunk, p.nchunks, sl2, lse, p.segs, raw);
    const int tiles = (N + kPoolTile - 1) / kPoolTile;
    hipLaunchKernelGGL(snap_pool, dim3((unsigned)(p.segs * tiles)), dim3(kPoolTile), 0, st, raw,
                       p.rgroups, p.segs, N, W, pool_k, tiles, score);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_snapkv(const void* q, const void* k, int dtype, int L, int B, int Hq, int Hkv,
                         int N, int W, int d, float scale, int pool_k, float* score, void* ws,
                         hipStream_t st) {
    if (dtype == 0) {
        if (d == 128) return run_snapkv<__bf16, 128>(q, k, L, B, Hq, Hkv, N, W, scale, pool_k, score, ws, st);
        return run_snapkv<__bf16, 64>(q, k, L, B, Hq, Hkv, N, W, scale, pool_k, score, ws, st);
    }
    if (d == 128) return run_snapkv<float, 128>(q, k, L, B, Hq, Hkv, N, W, scale, pool_k, score, ws, st);
    return run_snapkv<float, 64>(q, k, L, B, Hq, Hkv, N, W, scale, pool_k, score, ws, st);
}

}  // namespace kve
