// Per-role top-k selection (Algorithm 1, per-bucket top-k) with the window
// always kept, and the coalesced K/V compaction of the kept rows (§6: the
// dense cache of a compacting implementation).
//
// topk_select: one workgroup per (layer, sample, KV head) segment.  Scores are
// mapped to order-preserving 32-bit keys (-0 -> +0, NaN lowest) and, for every
// role bucket at once, a most-significant-digit radix select (4 passes of 8
// bits, one LDS histogram of 256 bins per bucket) finds the key of the
// quota-th largest candidate.  A final ordered pass keeps every key above the
// threshold and, among keys equal to it, the lowest indices first, and writes
// the kept positions in ascending order (ballot + prefix count per chunk).
#include "kve_device.h"
#include "kve_internal.h"

namespace kve {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kMaxR = 8;
constexpr int kDigits = 256;

enum : int { kModeNone = 0, kModeSelect = 1, kModeAll = 2 };

__global__ __launch_bounds__(kThreads) void topk_kernel(const float* __restrict__ score,
                                                        const int8_t* __restrict__ roles,
                                                        const int32_t* __restrict__ quota, int B,
                                                        int Hkv, int N, int W, int R, int k_cap,
                                                        int32_t* __restrict__ idx_out,
                                                        int32_t* __restrict__ count_out) {
    __shared__ uint32_t hist[kMaxR][kDigits];
    __shared__ uint32_t s_prefix[kMaxR];  // key bits fixed so far
    __shared__ int s_need[kMaxR];         // still to take among keys matching the prefix
    __shared__ int s_mode[kMaxR];
    __shared__ int s_wcnt[kWaves][kMaxR + 1];
    __shared__ int s_eq_seen[kMaxR];
    __shared__ int s_base;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int seg = blockIdx.x;
    const int b = (seg / Hkv) % B;
    const float* sc = score + (size_t)seg * N;
    const int8_t* ro = roles + (size_t)b * N;
    const int P = N - W;
    const uint64_t lt_mask = (1ull << lane) - 1ull;

    if (tid < R) {
        s_prefix[tid] = 0u;
        s_mode[tid] = kModeSelect;
        s_need[tid] = 0;
        s_eq_seen[tid] = 0;
    }
    if (tid == 0) s_base = 0;
    __syncthreads();

    for (int pass = 0; pass < 4; ++pass) {
        const int shift = 24 - 8 * pass;
        const uint32_t himask = pass == 0 ? 0u : (0xFFFFFFFFu << (shift + 8));
        for (int e = tid; e < R * kDigits; e += kThreads) hist[e / kDigits][e % kDigits] = 0u;
        __syncthreads();
        for (int t = tid; t < P; t += kThreads) {
            const int r = ro[t];
            if (r < 0 || r >= R || s_mode[r] != kModeSelect) continue;
            const uint32_t key = score_key(sc[t]);
            if ((key & himask) != s_prefix[r]) continue;
            atomicAdd(&hist[r][(key >> shift) & (kDigits - 1)], 1u);
        }
        __syncthreads();
        if (tid < R && s_mode[tid] == kModeSelect) {
            const int r = tid;
            if (pass == 0) {
                int n = 0;
                for (int dgt = 0; dgt < kDigits; ++dgt) n += (int)hist[r][dgt];
                const int q = max(quota[(size_t)b * R + r], 0);
                if (q == 0)
                    s_mode[r] = kModeNone;
                else if (q >= n)
                    s_mode[r] = kModeAll;
                else
                    s_need[r] = q;
            }
            if (s_mode[r] == kModeSelect) {
                const int want = s_need[r];
                int cum = 0, dgt = kDigits - 1;
                for (; dgt > 0; --dgt) {
                    const int hcount = (int)hist[r][dgt];
                    if (cum + hcount >= want) break;
                    cum += hcount;
                }
                s_prefix[r] |= (uint32_t)dgt << shift;
                s_need[r] = want - cum;
            }
        }
        __syncthreads();
    }

    // Ordered output pass: s_prefix[r] is the threshold key, s_need[r] >= 1 the
    // number of candidates equal to it that stay (lowest index first).
    for (int c0 = 0; c0 < N; c0 += kThreads) {
        const int t = c0 + tid;
        bool keep = false, eq = false;
        int r = -1;
        if (t < N) {
            if (t >= P) {
                keep = true;
            } else {
                r = ro[t];
                if (r >= 0 && r < R) {
                    const int mode = s_mode[r];
                    if (mode == kModeAll) {
                        keep = true;
                    } else if (mode == kModeSelect) {
                        const uint32_t key = score_key(sc[t]);
                        if (key > s_prefix[r])
                            keep = true;
                        else if (key == s_prefix[r])
                            eq = true;
                    }
                }
            }
        }
        int rank_w = 0;
        for (int rr = 0; rr < R; ++rr) {
            const bool mine = eq && r == rr;
            const uint64_t mask = __ballot(mine);
            if (mine) rank_w = __popcll(mask & lt_mask);
            if (lane == 0) s_wcnt[wave][rr] = __popcll(mask);
        }
        __syncthreads();
        if (eq) {
            int rank = s_eq_seen[r] + rank_w;
            for (int w = 0; w < wave; ++w) rank += s_wcnt[w][r];
            keep = rank < s_need[r];
        }
        const uint64_t km = __ballot(keep);
        if (lane == 0) s_wcnt[wave][kMaxR] = __popcll(km);
        __syncthreads();
        if (keep) {
            int pos = s_base + __popcll(km & lt_mask);
            for (int w = 0; w < wave; ++w) pos += s_wcnt[w][kMaxR];
            if (pos < k_cap) idx_out[(size_t)seg * k_cap + pos] = t;
        }
        __syncthreads();
        if (tid == 0) {
            int tot = 0;
            for (int w = 0; w < kWaves; ++w) tot += s_wcnt[w][kMaxR];
            s_base += tot;
        }
        if (tid < R) {
            int tot = 0;
            for (int w = 0; w < kWaves; ++w) tot += s_wcnt[w][tid];
            s_eq_seen[tid] += tot;
        }
        __syncthreads();
    }
    if (tid == 0 && count_out != nullptr) count_out[seg] = s_base;
}

constexpr int kCompactRows = 64;

__global__ __launch_bounds__(kThreads) void compact_kernel(const char* __restrict__ k,
                                                           const char* __restrict__ v, int row_bytes,
                                                           const int32_t* __restrict__ idx,
                                                           const int32_t* __restrict__ count, int N,
                                                           int k_cap, int nblk, char* __restrict__ k_out,
                                                           char* __restrict__ v_out) {
    const int blk = blockIdx.x % nblk;
    const int seg = blockIdx.x / nblk;
    const int cnt = min(count[seg], k_cap);
    const int m0 = blk * kCompactRows;
    if (m0 >= cnt) return;
    const int parts = row_bytes / 16;
    const int total = kCompactRows * parts;
    for (int e = threadIdx.x; e < total; e += kThreads) {
        const int mm = e / parts;
        const int part = e - mm * parts;
        const int m = m0 + mm;
        if (m >= cnt) break;
        const int t = idx[(size_t)seg * k_cap + m];
        if (t < 0 || t >= N) continue;
        const size_t src = ((size_t)seg * N + t) * row_bytes + (size_t)part * 16;
        const size_t dst = ((size_t)seg * k_cap + m) * row_bytes + (size_t)part * 16;
        st16(k_out + dst, ld16(k + src));
        if (v != nullptr) st16(v_out + dst, ld16(v + src));
    }
}

}  // namespace

hipError_t launch_topk(const float* score, const int8_t* roles, const int32_t* quota, int L, int B,
                       int Hkv, int N, int W, int R, int k_cap, int32_t* idx_out, int32_t* count_out,
                       hipStream_t st) {
    const size_t segs = (size_t)L * B * Hkv;
    hipLaunchKernelGGL(topk_kernel, dim3((unsigned)segs), dim3(kThreads), 0, st, score, roles, quota, B,
                       Hkv, N, W, R, k_cap, idx_out, count_out);
    return hipGetLastError();
}

hipError_t launch_compact(const void* k, const void* v, int elem_bytes, const int32_t* idx,
                          const int32_t* count, int L, int B, int Hkv, int N, int d, int k_cap,
                          void* k_out, void* v_out, hipStream_t st) {
    const size_t segs = (size_t)L * B * Hkv;
    const int nblk = (k_cap + kCompactRows - 1) / kCompactRows;
    if (nblk == 0 || segs == 0) return hipSuccess;
    hipLaunchKernelGGL(compact_kernel, dim3((unsigned)(segs * nblk)), dim3(kThreads), 0, st,
                       static_cast<const char*>(k), static_cast<const char*>(v), d * elem_bytes, idx,
                       count, N, k_cap, nblk, static_cast<char*>(k_out), static_cast<char*>(v_out));
    return hipGetLastError();
}

}  // namespace kve
