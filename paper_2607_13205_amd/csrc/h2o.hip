// H2O accumulated attention score, the baseline scorer.
//
// Paper §2 (H2O family): s(t) = sum over prefill queries i >= t of the causal
// softmax weight p_i(t), kept per (layer, head); here summed over the G query
// heads of each KV head.
//
// Both passes are the causal QK^T on the matrix cores (bf16 32x32x16, fp32
// 32x32x2) with operands streamed through a two-slot LDS ring by
// direct-to-LDS loads, as in the SnapKV kernels:
//   h2o_pass1  one workgroup per (KV group, block of positions): its 128 rows
//              are the G heads of the group at 128/G consecutive positions
//              (position-major), query fragments in registers; the keys up to
//              the block's last position stream through LDS and each lane
//              keeps one row's running softmax denominator.  Writes
//              -lse2/sl2 per row, the start value pass 2 needs, into rows of
//              pitch NP = N rounded up to 64 floats per head.
//   h2o_pass2  one workgroup per (query head, 128-key block), key blocks near
//              0 (the most rows) first: four waves own 32 keys each (key
//              fragments in registers); every later query row of the head
//              streams through LDS in 64-row chunks together with its
//              -lse2/sl2, which starts the products, so that sl2 * acc =
//              x - lse2 and each lane sums exp2 over its key's column
//              directly.  One column sum per (query head, key).
//   h2o_heads  adds the G heads of each KV group, in head order.
// Logits are in log2 units, x = scale * log2(e) * <q, k>.
#include <algorithm>

#include "kve_device.h"
#include "kve_internal.h"
#include "kve_stream.h"

namespace kve {
namespace {

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * 64;
constexpr int kKeys = 64;  // rows per chunk (keys in pass 1, query rows in pass 2)
// The operands are L2-resident: one chunk ahead suffices, and the smaller ring
// lets four workgroups share a compute unit.
constexpr int kRing = 2;
constexpr int kKeyBlock = 128;  // keys per pass-2 workgroup

template <typename T, int D>
struct Geo {
    using C = KChunk<T, D, kKeys>;
    using Rd = ChunkReader<T, D, kKeys>;
    using Wr = ChunkWriter<T, D, kKeys, kWaves>;
    using Ring = ChunkRing<T, D, kKeys, kWaves, kRing>;
    using Frags = typename Mma<T>::frag[C::NSTEP];
};

// Fragments of one row (key or query) of length D, zero when !valid.
template <typename T, int D>
__device__ __forceinline__ void load_row_frags(typename Geo<T, D>::Frags& f, const T* row, bool valid, int lane) {
    using M = Mma<T>;
#pragma unroll
    for (int st = 0; st < Geo<T, D>::C::NSTEP; ++st) {
        f[st] = valid ? M::load(row, st * M::KSTEP + (lane >> 5) * M::KPL) : M::zero();
        pin(f[st]);
    }
}

// Chunks of consecutive rows of one [N, D] matrix, from `first`.
template <typename T, int D>
struct RowChunks {
    const char* base;
    int first, end;
    __device__ __forceinline__ void operator()(int c, const char** rows, int* valid) const {
        const int r0 = first + c * kKeys;
        *rows = base + (size_t)r0 * Geo<T, D>::C::ROW;
        *valid = end - r0;
    }
};

template <typename T, int D>
__global__ __launch_bounds__(kThreads, 2) void h2o_pass1(const T* __restrict__ q, const T* __restrict__ k,
                                                         int Hq, int Hkv, int N, int NP, int npos, int nblk,
                                                         float sl2, float* __restrict__ linit) {
    using G = Geo<T, D>;
    __shared__ __align__(16) char ring[kRing * G::C::BYTES];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int Gh = Hq / Hkv;
    int bid = blockIdx.x;
    const int pb = nblk - 1 - bid % nblk;  // longest causal rows first
    bid /= nblk;
    const int j = bid % Hkv;
    const int lb = bid / Hkv;
    const int p0 = pb * npos;
    // this lane's row: head g of the group at position pos (position-major)
    const int r = wave * 32 + (lane & 31);
    const int g = r % Gh;
    const int pos = p0 + r / Gh;
    const bool valid = r < npos * Gh && pos < N;
    const size_t head = (size_t)lb * Hq + (size_t)j * Gh + g;

    typename G::Frags qf;
    load_row_frags<T, D>(qf, q + (head * N + (valid ? pos : 0)) * D, valid, lane);
    const int t_end = min(N, p0 + npos);  // keys up to the block's last position
    const int nch = (t_end + kKeys - 1) / kKeys;
    typename G::Rd rd;
    rd.init(lane, 0);
    typename G::Ring ring_io;
    ring_io.open(nch, wave, lane);
    const RowChunks<T, D> src{reinterpret_cast<const char*>(k) + ((size_t)lb * Hkv + j) * N * G::C::ROW, 0, t_end};
    ring_io.prologue(ring, src);

    const int lim = valid ? pos : -1;  // last key the row sees
    RowSum rs;
    for (int s0 = 0; s0 < nch; s0 += kRing) {
#pragma unroll
        for (int u = 0; u < kRing; ++u) {
            const int s = s0 + u;
            if (s >= nch) break;
            ring_io.advance(ring, s, u, src);
            f32x16 acc[2];
            chunk_mma<T, D, kKeys, true>(acc, rd, ring + u * G::C::BYTES, qf, nullptr, lane);
            if ((s + 1) * kKeys > p0) {  // a key of the chunk lies after some row of the block
                // key of element (kb, i) = base + 32 kb + 8 (i / 4) + i % 4
                const int last = lim - (s * kKeys + 4 * (lane >> 5));
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int i = 0; i < 16; ++i)
                        if (32 * kb + 8 * (i >> 2) + (i & 3) > last) acc[kb][i] = -INFINITY;
            }
            rs.add(acc, sl2);
        }
    }
    // the two lane halves hold the same row and different keys
    lse2_merge(rs.m, rs.l, __shfl_xor(rs.m, 32), __shfl_xor(rs.l, 32));
    if (lane < 32 && valid) linit[head * NP + pos] = -rs.lse2() / sl2;
}

template <typename T, int D>
__global__ __launch_bounds__(kThreads, 2) void h2o_pass2(const T* __restrict__ q, const T* __restrict__ k,
                                                         const float* __restrict__ linit, int heads, int Hq,
                                                         int Hkv, int N, int NP, float sl2,
                                                         float* __restrict__ colsum) {
    using G = Geo<T, D>;
    __shared__ __align__(16) char ring[kRing * G::C::BYTES];
    __shared__ __align__(16) float sli[kRing][kKeys];  // -lse2/sl2 of each chunk row
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int Gh = Hq / Hkv;
    const int kb = blockIdx.x / heads;  // key blocks near 0 (the most rows) first
    const size_t head = (size_t)(blockIdx.x - kb * heads);  // over all layers and samples
    const size_t lbj = head / Gh;                            // (layer, sample, KV head)
    const int kb0 = kb * kKeyBlock;
    const int key = kb0 + wave * 32 + (lane & 31);

    typename G::Frags kf;
    load_row_frags<T, D>(kf, k + (lbj * N + (key < N ? key : 0)) * D, key < N, lane);
    // rows kb0 .. N - 1 of this head
    const int nch = (N - kb0 + kKeys - 1) / kKeys;
    typename G::Rd rd;
    rd.init(lane, 0);
    typename G::Wr wr;
    wr.init(wave, lane);
    // chunk c: rows from kb0 + 64 c, with their 64 start values (256 bytes:
    // four 16-byte pieces per wave, lanes 0..3).  r0 is a multiple of 64 below
    // N, so the 64 values lie inside the head's row of pitch NP and start
    // 256-byte aligned; rows past N are masked.
    auto issue = [&](int c, int slot) {
        const int r0 = kb0 + c * kKeys;
        const char* rows = reinterpret_cast<const char*>(q) + (head * N + r0) * G::C::ROW;
        wr.issue(ring + slot * G::C::BYTES, rows, N - r0);
        if (lane < 4)
            lds_dma16(reinterpret_cast<const char*>(linit + head * NP + r0), (unsigned)(wave * 64 + lane * 16),
                      reinterpret_cast<const char*>(&sli[slot][wave * 16]));
    };
    for (int c = 0; c < min(kRing - 1, nch); ++c) issue(c, c);

    float col = 0.0f;
    for (int s0 = 0; s0 < nch; s0 += kRing) {
#pragma unroll
        for (int u = 0; u < kRing; ++u) {
            const int s = s0 + u;
            if (s >= nch) break;
            wait_chunk<G::Wr::LPW + 1, kRing - 2>(min(kRing - 2, nch - 1 - s));
            lds_barrier();
            if (s + kRing - 1 < nch) issue(s + kRing - 1, (u + kRing - 1) % kRing);
            f32x16 acc[2];
            chunk_mma<T, D, kKeys, true>(acc, rd, ring + u * G::C::BYTES, kf, &sli[u][0], lane);
            const int r0 = kb0 + s * kKeys;
            if (r0 < kb0 + kKeyBlock || r0 + kKeys > N) {  // rows before some key, or past N
                // row of element (b, i) = r0 + 32 b + 8 (i / 4) + 4 (lane / 32) + i % 4; it
                // counts iff key <= row < N
                const int lo = key - (r0 + 4 * (lane >> 5));
                const int hi = N - (r0 + 4 * (lane >> 5));
#pragma unroll
                for (int b = 0; b < 2; ++b)
#pragma unroll
                    for (int i = 0; i < 16; ++i) {
                        const int off = 32 * b + 8 * (i >> 2) + (i & 3);
                        if (off < lo || off >= hi) acc[b][i] = -INFINITY;
                    }
            }
            col += exp2_sum(acc, sl2);
        }
    }
    // the two lane halves hold the same key and different rows
    col += __shfl_xor(col, 32);
    if (lane < 32 && key < N) colsum[head * N + key] = col;
}

// score of (layer, sample, KV head j) = sum of its G heads' column sums, in head order
__global__ __launch_bounds__(kThreads) void h2o_heads(const float* __restrict__ colsum, int Gh, int N,
                                                      size_t total, float* __restrict__ score) {
    for (size_t e = (size_t)blockIdx.x * kThreads + threadIdx.x; e < total; e += (size_t)gridDim.x * kThreads) {
        const size_t lbj = e / N, t = e - lbj * N;
        const float* c = colsum + lbj * Gh * N + t;
        float v = 0.0f;
        for (int g = 0; g < Gh; ++g) v += c[(size_t)g * N];
        score[e] = v;
    }
}

template <typename T, int D>
hipError_t run_h2o(const void* q, const void* k, int L, int B, int Hq, int Hkv, int N, float scale,
                   float* score, void* ws, hipStream_t st) {
    float* linit = static_cast<float*>(ws);
    float* colsum = linit + h2o_colsum_offset(L, B, Hq, N);
    const float sl2 = scale * kLog2e;
    const T* qt = static_cast<const T*>(q);
    const T* kt = static_cast<const T*>(k);
    const int Gh = Hq / Hkv;
    const int npos = kH2oRowsPerGroup / Gh;  // positions per pass-1 workgroup
    const int nblk = (N + npos - 1) / npos;
    const int nkb = (N + kKeyBlock - 1) / kKeyBlock;
    const int NP = h2o_pitch(N);
    hipLaunchKernelGGL((h2o_pass1<T, D>), dim3((unsigned)((size_t)L * B * Hkv * nblk)), dim3(kThreads), 0, st, qt,
                       kt, Hq, Hkv, N, NP, npos, nblk, sl2, linit);
    const int heads = L * B * Hq;
    hipLaunchKernelGGL((h2o_pass2<T, D>), dim3((unsigned)((size_t)heads * nkb)), dim3(kThreads), 0, st, qt, kt,
                       linit, heads, Hq, Hkv, N, NP, sl2, colsum);
    const size_t total = (size_t)L * B * Hkv * N;
    hipLaunchKernelGGL(h2o_heads, dim3((unsigned)std::min<size_t>((total + kThreads - 1) / kThreads, 4096)),
                       dim3(kThreads), 0, st, colsum, Gh, N, total, score);
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
