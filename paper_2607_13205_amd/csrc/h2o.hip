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

// Start of the rows of head h of sample `lb` (layer * B + sample) in a view.
__device__ __forceinline__ const char* head_rows(const RowView& v, int lb, int B, int h) {
    return v.base + (long long)(lb / B) * v.s_layer + (long long)(lb % B) * v.s_batch + (long long)h * v.s_head;
}

// Fragments of one row (key or query) of length D, zero when !valid.
template <typename T, int D>
__device__ __forceinline__ void load_row_frags(typename Geo<T, D>::Frags& f, const char* row, bool valid, int lane) {
    using M = Mma<T>;
#pragma unroll
    for (int st = 0; st < Geo<T, D>::C::NSTEP; ++st) {
        f[st] = valid ? M::load(row, st * M::KSTEP + (lane >> 5) * M::KPL) : M::zero();
        pin(f[st]);
    }
}

// Chunks of consecutive rows of one [N, D] matrix (rows `stride` bytes
// apart), from `first`.
template <typename T, int D>
struct RowChunks {
    const char* base;
    long long stride;
    int first, end;
    __device__ __forceinline__ void operator()(int c, const char** rows, int* valid) const {
        const int r0 = first + c * kKeys;
        *rows = base + (long long)r0 * stride;
        *valid = end - r0;
    }
};

// Products of one chunk's first 64 rows (the A operand, from LDS) with two
// sets of 32 register rows: acc[s][b] is register set s against chunk block b
// (element i belongs to chunk row 32 b + c_row(i, lane), the lane to register
// row lane % 32 of set s).  Each fragment read from LDS feeds two products,
// and the four accumulators are independent chains.  Start values: zero, or
// init[chunk row] when given.
template <typename T, int D>
__device__ __forceinline__ void chunk_mma_x2(f32x16 (&acc)[2][2], const typename Geo<T, D>::Rd& rd,
                                             const char* slot, const typename Geo<T, D>::Frags& r0,
                                             const typename Geo<T, D>::Frags& r1, const float* init, int lane) {
    using M = Mma<T>;
    constexpr int NS = Geo<T, D>::C::NSTEP;
    f32x16 c0[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
        if (init == nullptr) {
            c0[b] = f32x16{};
        } else {
#pragma unroll
            for (int a = 0; a < 4; ++a) {
                const float4 v = *reinterpret_cast<const float4*>(init + 32 * b + c_row(4 * a, lane));
                c0[b][4 * a] = v.x;
                c0[b][4 * a + 1] = v.y;
                c0[b][4 * a + 2] = v.z;
                c0[b][4 * a + 3] = v.w;
            }
        }
    }
#pragma unroll
    for (int st = 0; st < NS; ++st) {
        const typename M::frag f[2] = {rd.get(slot, 0, st), rd.get(slot, 1, st)};
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            acc[0][b] = M::mma(f[b], r0[st], st == 0 ? c0[b] : acc[0][b]);
            acc[1][b] = M::mma(f[b], r1[st], st == 0 ? c0[b] : acc[1][b]);
        }
    }
    // keep the fragment reads two k-steps ahead of the products
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
    for (int st = 0; st < NS; ++st) {
        __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
        if (st + 2 < NS) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    }
}

// Pass 1 with two register row sets per wave (bf16): 256 rows per workgroup,
// the G heads of a KV group at 256/G consecutive positions, position-major;
// wave w holds rows 64 w .. 64 w + 63 as two sets of 32.
template <typename T, int D>
__global__ __launch_bounds__(kThreads, 2) void h2o_pass1_x2(RowView qv, RowView kv, int B, int Hq, int Hkv, int N,
                                                            int NP, int npos, int nblk, float sl2,
                                                            float* __restrict__ linit) {
    using G = Geo<T, D>;
    __shared__ __align__(16) char ring[kRing * G::C::BYTES];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int Gh = Hq / Hkv;
    // the KV head varies fastest: workgroups are dealt to the XCDs in turn, so
    // (with Hkv a divisor or multiple of their number) each XCD keeps to a few
    // heads and their key rows, re-read by every later position block, stay in
    // its L2; within a head the longest causal rows come first
    int bid = blockIdx.x;
    const int j = bid % Hkv;
    bid /= Hkv;
    const int pb = nblk - 1 - bid % nblk;
    const int lb = bid / nblk;
    const int p0 = pb * npos;
    int pos[2], lim[2];
    bool valid[2];
    size_t head[2];
    typename G::Frags qf[2];
#pragma unroll
    for (int rs = 0; rs < 2; ++rs) {
        const int r = wave * 64 + rs * 32 + (lane & 31);
        const int g = r % Gh;
        pos[rs] = p0 + r / Gh;
        valid[rs] = r < npos * Gh && pos[rs] < N;
        head[rs] = (size_t)lb * Hq + (size_t)j * Gh + g;
        load_row_frags<T, D>(qf[rs], head_rows(qv, lb, B, j * Gh + g) + (long long)(valid[rs] ? pos[rs] : 0) * qv.s_token,
                             valid[rs], lane);
        lim[rs] = valid[rs] ? pos[rs] : -1;  // last key the row sees
    }
    const int t_end = min(N, p0 + npos);  // keys up to the block's last position
    const int nch = (t_end + kKeys - 1) / kKeys;
    typename G::Rd rd;
    rd.init(lane, 0);
    typename G::Ring ring_io;
    ring_io.open(nch, wave, lane, (unsigned)kv.s_token);
    const RowChunks<T, D> src{head_rows(kv, lb, B, j), kv.s_token, 0, t_end};
    ring_io.prologue(ring, src);

    RowSum rsum[2];
    for (int s0 = 0; s0 < nch; s0 += kRing) {
#pragma unroll
        for (int u = 0; u < kRing; ++u) {
            const int s = s0 + u;
            if (s >= nch) break;
            ring_io.advance(ring, s, u, src);
            f32x16 acc[2][2];
            chunk_mma_x2<T, D>(acc, rd, ring + u * G::C::BYTES, qf[0], qf[1], nullptr, lane);
            if ((s + 1) * kKeys > p0) {  // a key of the chunk lies after some row of the block
#pragma unroll
                for (int rs = 0; rs < 2; ++rs) {
                    // key of element (kb, i) = base + 32 kb + 8 (i / 4) + i % 4
                    const int last = lim[rs] - (s * kKeys + 4 * (lane >> 5));
#pragma unroll
                    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                        for (int i = 0; i < 16; ++i)
                            if (32 * kb + 8 * (i >> 2) + (i & 3) > last) acc[rs][kb][i] = -INFINITY;
                }
            }
            row_sums_add<2>(rsum, acc, sl2);
        }
    }
#pragma unroll
    for (int rs = 0; rs < 2; ++rs) {
        // the two lane halves hold the same row and different keys
        lse2_merge(rsum[rs].m, rsum[rs].l, __shfl_xor(rsum[rs].m, 32), __shfl_xor(rsum[rs].l, 32));
        if (lane < 32 && valid[rs]) linit[head[rs] * NP + pos[rs]] = -rsum[rs].lse2() / sl2;
    }
}

template <typename T, int D>
__global__ __launch_bounds__(kThreads, 2) void h2o_pass1(RowView qv, RowView kv, int B, int Hq, int Hkv, int N,
                                                         int NP, int npos, int nblk, float sl2,
                                                         float* __restrict__ linit) {
    using G = Geo<T, D>;
    __shared__ __align__(16) char ring[kRing * G::C::BYTES];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int Gh = Hq / Hkv;
    // the KV head varies fastest: workgroups are dealt to the XCDs in turn, so
    // (with Hkv a divisor or multiple of their number) each XCD keeps to a few
    // heads and their key rows, re-read by every later position block, stay in
    // its L2; within a head the longest causal rows come first
    int bid = blockIdx.x;
    const int j = bid % Hkv;
    bid /= Hkv;
    const int pb = nblk - 1 - bid % nblk;
    const int lb = bid / nblk;
    const int p0 = pb * npos;
    // this lane's row: head g of the group at position pos (position-major)
    const int r = wave * 32 + (lane & 31);
    const int g = r % Gh;
    const int pos = p0 + r / Gh;
    const bool valid = r < npos * Gh && pos < N;
    const size_t head = (size_t)lb * Hq + (size_t)j * Gh + g;

    typename G::Frags qf;
    load_row_frags<T, D>(qf, head_rows(qv, lb, B, j * Gh + g) + (long long)(valid ? pos : 0) * qv.s_token, valid,
                         lane);
    const int t_end = min(N, p0 + npos);  // keys up to the block's last position
    const int nch = (t_end + kKeys - 1) / kKeys;
    typename G::Rd rd;
    rd.init(lane, 0);
    typename G::Ring ring_io;
    ring_io.open(nch, wave, lane, (unsigned)kv.s_token);
    const RowChunks<T, D> src{head_rows(kv, lb, B, j), kv.s_token, 0, t_end};
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
__global__ __launch_bounds__(kThreads, 2) void h2o_pass2(RowView qv, RowView kv, int B,
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
    const char* qhead = head_rows(qv, (int)(head / Hq), B, (int)(head % Hq));
    load_row_frags<T, D>(kf, head_rows(kv, (int)(lbj / Hkv), B, (int)(lbj % Hkv)) + (long long)(key < N ? key : 0) * kv.s_token,
                         key < N, lane);
    // rows kb0 .. N - 1 of this head
    const int nch = (N - kb0 + kKeys - 1) / kKeys;
    typename G::Rd rd;
    rd.init(lane, 0);
    typename G::Wr wr;
    wr.init(wave, lane, (unsigned)qv.s_token);
    // chunk c: rows from kb0 + 64 c, with their 64 start values (256 bytes:
    // four 16-byte pieces per wave, lanes 0..3).  r0 is a multiple of 64 below
    // N, so the 64 values lie inside the head's row of pitch NP and start
    // 256-byte aligned; rows past N are masked.
    auto issue = [&](int c, int slot) {
        const int r0 = kb0 + c * kKeys;
        const char* rows = qhead + (long long)r0 * qv.s_token;
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

// Pass 2 with two register key sets per wave (bf16): 256 keys per workgroup,
// wave w holding keys 64 w .. 64 w + 63 as two sets of 32; every chunk of
// query rows read from LDS feeds both sets.
template <typename T, int D>
__global__ __launch_bounds__(kThreads, 2) void h2o_pass2_x2(RowView qv, RowView kv, int B,
                                                            const float* __restrict__ linit, int heads, int Hq,
                                                            int Hkv, int N, int NP, float sl2,
                                                            float* __restrict__ colsum) {
    using G = Geo<T, D>;
    constexpr int kBlock = 2 * kKeyBlock;
    __shared__ __align__(16) char ring[kRing * G::C::BYTES];
    __shared__ __align__(16) float sli[kRing][kKeys];  // -lse2/sl2 of each chunk row
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int Gh = Hq / Hkv;
    const int kb = blockIdx.x / heads;  // key blocks near 0 (the most rows) first
    const size_t head = (size_t)(blockIdx.x - kb * heads);  // over all layers and samples
    const size_t lbj = head / Gh;                            // (layer, sample, KV head)
    const int kb0 = kb * kBlock;
    int key[2];
    typename G::Frags kf[2];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
        key[ks] = kb0 + wave * 64 + ks * 32 + (lane & 31);
        load_row_frags<T, D>(kf[ks],
                             head_rows(kv, (int)(lbj / Hkv), B, (int)(lbj % Hkv)) +
                                 (long long)(key[ks] < N ? key[ks] : 0) * kv.s_token,
                             key[ks] < N, lane);
    }
    const char* qhead = head_rows(qv, (int)(head / Hq), B, (int)(head % Hq));
    // rows kb0 .. N - 1 of this head
    const int nch = (N - kb0 + kKeys - 1) / kKeys;
    typename G::Rd rd;
    rd.init(lane, 0);
    typename G::Wr wr;
    wr.init(wave, lane, (unsigned)qv.s_token);
    // chunk c: rows from kb0 + 64 c, with their 64 start values (256 bytes:
    // four 16-byte pieces per wave, lanes 0..3); as in h2o_pass2
    auto issue = [&](int c, int slot) {
        const int r0 = kb0 + c * kKeys;
        const char* rows = qhead + (long long)r0 * qv.s_token;
        wr.issue(ring + slot * G::C::BYTES, rows, N - r0);
        if (lane < 4)
            lds_dma16(reinterpret_cast<const char*>(linit + head * NP + r0), (unsigned)(wave * 64 + lane * 16),
                      reinterpret_cast<const char*>(&sli[slot][wave * 16]));
    };
    for (int c = 0; c < min(kRing - 1, nch); ++c) issue(c, c);

    float col[2] = {0.0f, 0.0f};
    for (int s0 = 0; s0 < nch; s0 += kRing) {
#pragma unroll
        for (int u = 0; u < kRing; ++u) {
            const int s = s0 + u;
            if (s >= nch) break;
            wait_chunk<G::Wr::LPW + 1, kRing - 2>(min(kRing - 2, nch - 1 - s));
            lds_barrier();
            if (s + kRing - 1 < nch) issue(s + kRing - 1, (u + kRing - 1) % kRing);
            f32x16 acc[2][2];
            chunk_mma_x2<T, D>(acc, rd, ring + u * G::C::BYTES, kf[0], kf[1], &sli[u][0], lane);
            const int r0 = kb0 + s * kKeys;
            if (r0 < kb0 + kBlock || r0 + kKeys > N) {  // rows before some key, or past N
#pragma unroll
                for (int ks = 0; ks < 2; ++ks) {
                    // row of element (b, i) = r0 + 32 b + 8 (i / 4) + 4 (lane / 32) + i % 4; it
                    // counts iff key <= row < N
                    const int lo = key[ks] - (r0 + 4 * (lane >> 5));
                    const int hi = N - (r0 + 4 * (lane >> 5));
#pragma unroll
                    for (int b = 0; b < 2; ++b)
#pragma unroll
                        for (int i = 0; i < 16; ++i) {
                            const int off = 32 * b + 8 * (i >> 2) + (i & 3);
                            if (off < lo || off >= hi) acc[ks][b][i] = -INFINITY;
                        }
                }
            }
            col[0] += exp2_sum(acc[0], sl2);
            col[1] += exp2_sum(acc[1], sl2);
        }
    }
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
        // the two lane halves hold the same key and different rows
        const float c = col[ks] + __shfl_xor(col[ks], 32);
        if (lane < 32 && key[ks] < N) colsum[head * N + key[ks]] = c;
    }
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
hipError_t run_h2o(const RowView& qv, const RowView& kv, int L, int B, int Hq, int Hkv, int N, float scale,
                   float* score, void* ws, hipStream_t st) {
    float* linit = static_cast<float*>(ws);
    float* colsum = linit + h2o_colsum_offset(L, B, Hq, N);
    const float sl2 = scale * kLog2e;
    const int Gh = Hq / Hkv;
    const int NP = h2o_pitch(N);
    const int heads = L * B * Hq;
    // bf16: two register row sets per wave (fp32 fragments are twice the
    // registers and keep one)
    constexpr bool kX2 = sizeof(T) == 2;
    const int npos = (kX2 ? 2 : 1) * kH2oRowsPerGroup / Gh;  // positions per pass-1 workgroup
    const int nblk = (N + npos - 1) / npos;
    const int kblock = (kX2 ? 2 : 1) * kKeyBlock;
    const int nkb = (N + kblock - 1) / kblock;
    if constexpr (kX2) {
        hipLaunchKernelGGL((h2o_pass1_x2<T, D>), dim3((unsigned)((size_t)L * B * Hkv * nblk)), dim3(kThreads), 0,
                           st, qv, kv, B, Hq, Hkv, N, NP, npos, nblk, sl2, linit);
        hipLaunchKernelGGL((h2o_pass2_x2<T, D>), dim3((unsigned)((size_t)heads * nkb)), dim3(kThreads), 0, st, qv,
                           kv, B, linit, heads, Hq, Hkv, N, NP, sl2, colsum);
    } else {
        hipLaunchKernelGGL((h2o_pass1<T, D>), dim3((unsigned)((size_t)L * B * Hkv * nblk)), dim3(kThreads), 0, st,
                           qv, kv, B, Hq, Hkv, N, NP, npos, nblk, sl2, linit);
        hipLaunchKernelGGL((h2o_pass2<T, D>), dim3((unsigned)((size_t)heads * nkb)), dim3(kThreads), 0, st, qv,
                           kv, B, linit, heads, Hq, Hkv, N, NP, sl2, colsum);
    }
    const size_t total = (size_t)L * B * Hkv * N;
    hipLaunchKernelGGL(h2o_heads, dim3((unsigned)std::min<size_t>((total + kThreads - 1) / kThreads, 4096)),
                       dim3(kThreads), 0, st, colsum, Gh, N, total, score);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_h2o(const RowView& q, const RowView& k, int dtype, int L, int B, int Hq, int Hkv, int N,
                      int d, float scale, float* score, void* ws, hipStream_t st) {
    if (dtype == 0) {
        if (d == 128) return run_h2o<__bf16, 128>(q, k, L, B, Hq, Hkv, N, scale, score, ws, st);
        return run_h2o<__bf16, 64>(q, k, L, B, Hq, Hkv, N, scale, score, ws, st);
    }
    if (d == 128) return run_h2o<float, 128>(q, k, L, B, Hq, Hkv, N, scale, score, ws, st);
    return run_h2o<float, 64>(q, k, L, B, Hq, Hkv, N, scale, score, ws, st);
}

}  // namespace kve
