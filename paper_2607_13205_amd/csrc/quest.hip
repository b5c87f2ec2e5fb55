// One-shot Quest analogue (§4.1 "Query-aware baseline"): the candidate prefix
// of every segment (layer, sample, KV head) is cut into pages of `page`
// consecutive tokens (the last one ragged; the window belongs to no page).
// A page's score is Quest's key bound: per head h of the group, the sum over
// channels of max(qbar_h[c] kmin[c], qbar_h[c] kmax[c]), with kmin and kmax the
// per-channel extremes of the page's keys and qbar_h the mean of head h's
// window queries, summed over the group's heads.  Every prefix token gets its
// page's score and the window +inf, so that the per-bucket top-k keeps whole
// pages in bound order.
//
// One pass over K: a group of lanes covers one key row (16 bytes each), so a
// wave streams several pages side by side, keeping running per-channel minima
// and maxima in registers; the bound is then a short reduction over the group.
// HBM-bound: K is read once, one float written per token.
#include "kve_device.h"
#include "kve_internal.h"

namespace kve {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kRowBatch = 16;  // key rows loaded before any is used

// Start of the rows of head `h` of segment seg's (layer, sample) in a view:
// segments are (layer, sample, KV head), KV head fastest.
__device__ __forceinline__ const char* seg_head_rows(const RowView& v, int seg, int B, int Hkv, int h) {
    const int lb = seg / Hkv;
    return v.base + (long long)(lb / B) * v.s_layer + (long long)(lb % B) * v.s_batch + (long long)h * v.s_head;
}

// qbar[seg, h, c] = mean over the W window rows of head h (float32).  A thread
// takes one 16-byte piece of a row (CW channels) of one head and adds the W
// rows in order, eight rows' loads in flight at a time.
template <typename T>
__global__ __launch_bounds__(kThreads) void quest_qmean(RowView qv, int B, int Hkv, int W, int G, int D,
                                                        float* __restrict__ qbar) {
    using VP = VPiece<T>;
    constexpr int CW = VP::CW;
    constexpr int kBatch = 8;
    const int seg = blockIdx.x;
    const float inv = 1.0f / (float)W;
    const int pieces = D / CW;  // per row
    for (int e = threadIdx.x; e < G * pieces; e += kThreads) {
        const int h = e / pieces, pc = e - (e / pieces) * pieces;
        const char* rows = seg_head_rows(qv, seg, B, Hkv, (seg % Hkv) * G + h) + (long long)pc * 16;
        float acc[CW] = {};
        int i = 0;
        for (; i + kBatch <= W; i += kBatch) {
            u32x4 raw[kBatch];
#pragma unroll
            for (int j = 0; j < kBatch; ++j) raw[j] = ld16(rows + (long long)(i + j) * qv.s_token);
#pragma unroll
            for (int j = 0; j < kBatch; ++j) {
                float f[CW];
                VP::to_f(raw[j], f);
#pragma unroll
                for (int c = 0; c < CW; ++c) acc[c] += f[c];
            }
        }
        for (; i < W; ++i) {
            float f[CW];
            VP::to_f(ld16(rows + (long long)i * qv.s_token), f);
#pragma unroll
            for (int c = 0; c < CW; ++c) acc[c] += f[c];
        }
        float* dst = qbar + (size_t)seg * G * D + (size_t)h * D + (size_t)pc * CW;
#pragma unroll
        for (int c = 0; c < CW; ++c) dst[c] = acc[c] * inv;
    }
}

// One workgroup per (segment, range of pages).  NH: heads per KV head padded
// to 4 or 8 (the padded heads have a zero mean query and add nothing).
template <typename T, int D, int NH>
__global__ __launch_bounds__(kThreads) void quest_pages(RowView kv, int B, int Hkv, const float* __restrict__ qbar,
                                                        int N, int W, int G, int page, int n_pages, int nranges,
                                                        int range_pages, float* __restrict__ score) {
    using VP = VPiece<T>;
    constexpr int CW = VP::CW;        // channels per lane
    constexpr int CPL = D / CW;       // lanes per key row
    constexpr int PPW = kWave / CPL;  // pages per wave step
    static_assert(NH == 4 || NH == 8, "4 or 8 padded heads");

    const int seg = blockIdx.x / nranges;
    const int rg = blockIdx.x - seg * nranges;
    const int lane = threadIdx.x & (kWave - 1);
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int grp = lane / CPL, cg = lane - (lane / CPL) * CPL;
    const int P = N - W;
    float* srow = score + (size_t)seg * N;

    if (rg == 0)
        for (int e = threadIdx.x; e < W; e += kThreads) srow[P + e] = INFINITY;

    // this lane's channels of every head's mean query
    float qv[NH][CW];
#pragma unroll
    for (int h = 0; h < NH; ++h)
#pragma unroll
        for (int c = 0; c < CW; ++c) qv[h][c] = h < G ? qbar[((size_t)seg * G + h) * D + cg * CW + c] : 0.0f;

    const char* ks = seg_head_rows(kv, seg, B, Hkv, seg % Hkv) + (long long)cg * CW * sizeof(T);
    const int p0 = rg * range_pages, p1 = min(n_pages, p0 + range_pages);
    for (int base = p0 + wv * PPW; base < p1; base += kWaves * PPW) {
        const int pg = min(base + grp, p1 - 1);  // groups past the range redo the last page, unwritten
        const int t0 = pg * page, t1 = min(t0 + page, P);
        float kmin[CW], kmax[CW];
#pragma unroll
        for (int c = 0; c < CW; ++c) {
            kmin[c] = INFINITY;
            kmax[c] = -INFINITY;
        }
        // rows past a ragged last page repeat its last row: extremes unchanged
        const char* pbase = ks + (long long)t0 * kv.s_token;
        const int last = t1 - t0 - 1;
        for (int r0 = 0; r0 < page; r0 += kRowBatch) {
            // every load of the batch in flight before the first is used;
            // non-temporal: each key row is read once
            u32x4 raw[kRowBatch];
#pragma unroll
            for (int i = 0; i < kRowBatch; ++i)
                raw[i] = __builtin_nontemporal_load(
                    reinterpret_cast<const u32x4*>(pbase + (long long)min(r0 + i, last) * kv.s_token));
#pragma unroll
            for (int i = 0; i < kRowBatch; i += 2) {
                float fa[CW], fb[CW];
                VP::to_f(raw[i], fa);
                VP::to_f(raw[i + 1], fb);
#pragma unroll
                for (int c = 0; c < CW; ++c) {  // three-input minimum and maximum: two rows per step
                    kmin[c] = fminf(fminf(kmin[c], fa[c]), fb[c]);
                    kmax[c] = fmaxf(fmaxf(kmax[c], fa[c]), fb[c]);
                }
            }
        }
        float s = 0.0f;
#pragma unroll
        for (int h = 0; h < NH; ++h)
#pragma unroll
            for (int c = 0; c < CW; ++c) s += fmaxf(qv[h][c] * kmin[c], qv[h][c] * kmax[c]);
#pragma unroll
        for (int m = 1; m < CPL; m <<= 1) s += __shfl_xor(s, m);
        if (base + grp < p1)
            for (int e = cg; e < t1 - t0; e += CPL) srow[t0 + e] = s;
    }
}

template <typename T, int D, int NH>
hipError_t run_quest(const RowView& q, const RowView& k, int L, int B, int Hq, int Hkv, int N, int W, int page,
                     float* score, void* ws, hipStream_t st) {
    const QuestPlan p = quest_plan(L, B, Hq, Hkv, N, W, D, (int)sizeof(T), page);
    float* qbar = static_cast<float*>(ws);
    hipLaunchKernelGGL((quest_qmean<T>), dim3((unsigned)p.segs), dim3(kThreads), 0, st, q, B, Hkv, W, p.G, D, qbar);
    hipLaunchKernelGGL((quest_pages<T, D, NH>), dim3((unsigned)((size_t)p.segs * p.nranges)), dim3(kThreads), 0, st,
                       k, B, Hkv, qbar, N, W, p.G, page, p.n_pages, p.nranges, p.range_pages, score);
    return hipGetLastError();
}

template <typename T, int D>
hipError_t run_quest_g(const RowView& q, const RowView& k, int L, int B, int Hq, int Hkv, int N, int W, int page,
                       float* score, void* ws, hipStream_t st) {
    if (Hq / Hkv <= 4) return run_quest<T, D, 4>(q, k, L, B, Hq, Hkv, N, W, page, score, ws, st);
    return run_quest<T, D, 8>(q, k, L, B, Hq, Hkv, N, W, page, score, ws, st);
}

}  // namespace

hipError_t launch_quest(const RowView& q, const RowView& k, int dtype, int L, int B, int Hq, int Hkv, int N, int W,
                        int d, int page, float* score, void* ws, hipStream_t st) {
    if (dtype == 0) {
        if (d == 128) return run_quest_g<__bf16, 128>(q, k, L, B, Hq, Hkv, N, W, page, score, ws, st);
        return run_quest_g<__bf16, 64>(q, k, L, B, Hq, Hkv, N, W, page, score, ws, st);
    }
    if (d == 128) return run_quest_g<float, 128>(q, k, L, B, Hq, Hkv, N, W, page, score, ws, st);
    return run_quest_g<float, 64>(q, k, L, B, Hq, Hkv, N, W, page, score, ws, st);
}

}  // namespace kve
