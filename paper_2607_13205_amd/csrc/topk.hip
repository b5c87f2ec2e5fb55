// Per-role top-k selection (Algorithm 1, per-bucket top-k) with the window
// always kept, and the coalesced K/V compaction of the kept rows (§6: the
// dense cache of a compacting implementation).
//
// topk_select: one workgroup per (layer, sample, KV head) segment.  Scores are
// mapped to order-preserving 32-bit keys (-0 -> +0, NaN lowest).
//   1. Three most-significant-digit passes (11, 11 and 10 bits), all buckets
//      at once with one LDS histogram per bucket, fix the key of the quota-th
//      largest candidate (the threshold) and how many candidates equal to it
//      stay.  The first digit holds the sign and all exponent bits, so float
//      scores spread over its bins; the first histogram also gives each
//      bucket's population, which decides whether the bucket is kept whole,
//      skipped, or selected.  The digit is found by all threads at once (a
//      scan over groups of bins).
//   2. Each wave owns a contiguous quarter of the positions and walks it 64
//      positions at a time: per-lane counts give what each wave run keeps
//      (keys above the threshold, the window, whole buckets, and keys equal to
//      the threshold lowest index first); ballots then rank the kept positions
//      so that they come out in ascending order.
// The sweeps read 16 positions per thread before they use any, so that the
// memory latency is paid once per group and not once per key; the loads are
// unconditional (clamped to a valid position) so that none waits behind a
// branch.
#include <type_traits>

#include "kve_device.h"
#include "kve_internal.h"

namespace kve {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kMaxR = 8;  // buckets supported (one kernel instantiation each)
constexpr int kDigitBits = 11;
constexpr int kDigits = 1 << kDigitBits;
constexpr int kBatch = 16;

enum : int { kModeNone = 0, kModeSelect = 1, kModeAll = 2 };

template <int R>
struct TopkShared {
    uint32_t hist[R][kDigits];
    uint32_t pref[R];  // key bits fixed so far (bits lo .. 31)
    int lo[R];         // lowest fixed bit; 0 once the threshold is known
    int need[R];       // still to take among keys matching the prefix
    int mode[R];
    int wave_eq[kWaves][R];  // equal-to-threshold candidates per wave run
    int wave_keep[kWaves];       // kept positions per wave run
    int scan[kWaves];
};

// Exclusive prefix sum over the workgroup of one value per thread (in thread
// order); every thread also gets the total.  `tmp` holds kWaves ints.
__device__ __forceinline__ int block_exclusive_scan(int v, int* tmp, int& total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int incl = v;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const int o = __shfl_up(incl, off);
        if (lane >= off) incl += o;
    }
    if (lane == kWave - 1) tmp[wave] = incl;
    __syncthreads();
    int before = 0;
    total = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
        const int t = tmp[w];
        if (w < wave) before += t;
        total += t;
    }
    __syncthreads();
    return before + incl - v;
}

template <int R>
__global__ __launch_bounds__(kThreads) void topk_kernel(const float* __restrict__ score,
                                                        const int8_t* __restrict__ roles,
                                                        const int32_t* __restrict__ quota, int B,
                                                        int Hkv, int N, int W, int k_cap,
                                                        int32_t* __restrict__ idx_out,
                                                        int32_t* __restrict__ count_out) {
    __shared__ TopkShared<R> sh;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int seg = blockIdx.x;
    const int b = (seg / Hkv) % B;
    const float* sc = score + (size_t)seg * N;
    const int8_t* ro = roles + (size_t)b * N;
    const int P = N - W;

    if (tid < R) {
        sh.mode[tid] = kModeSelect;  // decided after the first histogram
        sh.pref[tid] = 0u;
        sh.lo[tid] = 32;
        sh.need[tid] = 0;
    }
    __syncthreads();

    // 1. radix passes over the keys, all buckets at once: digits of 11, 11 and
    //    10 bits from the top; the first covers the sign and exponent bits
    for (int pass = 0; pass < (32 + kDigitBits - 1) / kDigitBits; ++pass) {
        bool any = false;
#pragma unroll
        for (int r = 0; r < R; ++r) any |= sh.mode[r] == kModeSelect && sh.lo[r] > 0;
        if (!any) break;  // uniform: every thread reads the same LDS values
        for (int e = tid; e < R * kDigits; e += kThreads) (&sh.hist[0][0])[e] = 0u;
        __syncthreads();
        // every bucket's state in registers; a key is counted when it matches
        // its bucket's prefix, the bucket picked with selects (no branches)
        bool act[R];
        uint32_t pf[R];
        int lov[R];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            act[r] = sh.mode[r] == kModeSelect && sh.lo[r] > 0;
            pf[r] = sh.pref[r];
            lov[r] = sh.lo[r];
        }
        // the first pass counts every labelled candidate on its top digit (no
        // prefix yet, every bucket still selecting); the later ones only the
        // keys that match their bucket's prefix
        auto count_keys = [&](auto first) {
            for (int t00 = tid; t00 < P; t00 += kThreads * kBatch) {
                int rv[kBatch];
                float sv[kBatch];
#pragma unroll
                for (int e = 0; e < kBatch; ++e) {  // unconditional loads (clamped index), then the bound
                    const int t = t00 + e * kThreads;
                    const int tc = min(t, P - 1);
                    const int r = ro[tc];
                    sv[e] = sc[tc];
                    rv[e] = t < P ? r : -1;
                }
#pragma unroll
                for (int e = 0; e < kBatch; ++e) {
                    const int r = rv[e];
                    const uint32_t key = score_key(sv[e]);
                    if constexpr (decltype(first)::value) {
                        if ((unsigned)r < (unsigned)R) atomicAdd(&sh.hist[r][key >> (32 - kDigitBits)], 1u);
                    } else {
                        bool a = false;
                        uint32_t p = 0u;
                        int lo = 32;
#pragma unroll
                        for (int q = 0; q < R; ++q) {
                            a = r == q ? act[q] : a;
                            p = r == q ? pf[q] : p;
                            lo = r == q ? lov[q] : lo;
                        }
                        a = a && (lo >= 32 || (key >> lo) == p);
                        const int w = min(kDigitBits, lo);
                        if (a) atomicAdd(&sh.hist[r][(key >> (lo - w)) & ((1u << w) - 1u)], 1u);
                    }
                }
            }
        };
        if (pass == 0)
            count_keys(std::true_type{});
        else
            count_keys(std::false_type{});
        __syncthreads();
        // Digit search, every thread at once: thread tid holds the kPerThread
        // bins from the top going down; a scan gives the count of keys in all
        // higher bins, and the thread whose bins reach `want` finds the digit.
        // After the first histogram (the bucket's whole population) the bucket
        // is kept whole, skipped, or selected.
#pragma unroll 1
        for (int r = 0; r < R; ++r) {
            if (!(sh.mode[r] == kModeSelect && sh.lo[r] > 0)) continue;  // uniform
            constexpr int kPerThread = kDigits / kThreads;
            const int hi = kDigits - kPerThread * tid;  // bins [hi - kPerThread, hi)
            int mine = 0;
#pragma unroll
            for (int e = 1; e <= kPerThread; ++e) mine += (int)sh.hist[r][hi - e];
            int total;
            const int above = block_exclusive_scan(mine, sh.scan, total);
            int want = sh.need[r];
            if (pass == 0) {
                const int q = max(quota[(size_t)b * R + r], 0);
                if (q == 0 || q >= total) {
                    if (tid == 0) sh.mode[r] = q == 0 ? kModeNone : kModeAll;
                    __syncthreads();
                    continue;
                }
                want = q;
            }
            if (above < want && above + mine >= want) {  // exactly one thread
                const int lo = sh.lo[r], w = min(kDigitBits, lo);
                int cum = above, dgt = hi - 1;
                for (; dgt > hi - kPerThread; --dgt) {
                    const int h = (int)sh.hist[r][dgt];
                    if (cum + h >= want) break;
                    cum += h;
                }
                sh.pref[r] = (lo < 32 ? sh.pref[r] << w : 0u) | (uint32_t)dgt;
                sh.need[r] = want - cum;
                sh.lo[r] = lo - w;
            }
            __syncthreads();
        }
    }

    // 2. ordered output over wave runs [w0, w1), 64 positions per step
    int mode[R], need[R];
    uint32_t th[R];  // threshold key of each selecting bucket
#pragma unroll
    for (int r = 0; r < R; ++r) {
        mode[r] = sh.mode[r];
        th[r] = sh.pref[r];
        need[r] = mode[r] == kModeSelect ? sh.need[r] : 0;
    }
    const int run = (N + kWaves * kWave - 1) / (kWaves * kWave) * kWave;  // positions per wave, whole steps
    const int w0 = min(N, wave * run), w1 = min(N, w0 + run);
    // class of position t: 1 kept, 2 + r equal to the threshold of bucket r, 0
    // dropped; the bucket's mode and threshold are picked with selects (a
    // branch per bucket would cost every key a divergent branch)
    auto classify = [&](int t, int r, float x) {
        int m = kModeNone;
        uint32_t thr = 0u;
#pragma unroll
        for (int q = 0; q < R; ++q) {
            m = r == q ? mode[q] : m;
            thr = r == q ? th[q] : thr;
        }
        const uint32_t key = score_key(x);
        const int sel = key > thr ? 1 : (key == thr ? 2 + r : 0);
        const int c = m == kModeAll ? 1 : (m == kModeSelect ? sel : 0);
        return t >= P ? 1 : c;
    };
    // visit(t, c) for every position of this wave's run, 64 consecutive per step
    auto sweep = [&](auto&& visit) {
        for (int s00 = w0; s00 < w1; s00 += kWave * kBatch) {
            int rv[kBatch];
            float sv[kBatch];
#pragma unroll
            for (int e = 0; e < kBatch; ++e) {  // unconditional loads (clamped index), then the bound
                const int t = s00 + e * kWave + lane;
                const int tc = max(0, min(t, min(w1, P) - 1));
                const int r = ro[tc];
                sv[e] = sc[tc];
                rv[e] = t < min(w1, P) ? r : -1;
            }
#pragma unroll
            for (int e = 0; e < kBatch; ++e) {
                const int t = s00 + e * kWave + lane;
                visit(t, t < w1 ? classify(t, rv[e], sv[e]) : 0);
            }
        }
    };
    const uint64_t lt = (1ull << lane) - 1ull;
    // count this run's kept positions and its equal keys per bucket, per lane,
    // then over the wave
    int keep = 0, eq[R];
#pragma unroll
    for (int r = 0; r < R; ++r) eq[r] = 0;
    sweep([&](int, int c) {
        keep += c == 1;
#pragma unroll
        for (int r = 0; r < R; ++r) eq[r] += c == 2 + r;
    });
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        keep += __shfl_xor(keep, off);
#pragma unroll
        for (int r = 0; r < R; ++r) eq[r] += __shfl_xor(eq[r], off);
    }
    if (lane == 0) {
#pragma unroll
        for (int r = 0; r < R; ++r) sh.wave_eq[wave][r] = eq[r];
    }
    __syncthreads();
    // equal keys are kept lowest index first: the earlier runs' equal keys come first
    int eq_seen[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        eq_seen[r] = 0;
        for (int w = 0; w < wave; ++w) eq_seen[r] += sh.wave_eq[w][r];
        keep += max(0, min(eq[r], need[r] - eq_seen[r]));
    }
    if (lane == 0) sh.wave_keep[wave] = keep;
    __syncthreads();
    int pos = 0, total = 0;
    for (int w = 0; w < kWaves; ++w) {
        if (w < wave) pos += sh.wave_keep[w];
        total += sh.wave_keep[w];
    }
    sweep([&](int t, int c) {
        bool k = c == 1;
        if (__ballot(c >= 2) != 0ull) {  // rare: keys equal to a threshold in this step
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const uint64_t m = __ballot(c == 2 + r);
                if (c == 2 + r) k = eq_seen[r] + __popcll(m & lt) < need[r];
                eq_seen[r] += __popcll(m);
            }
        }
        const uint64_t km = __ballot(k);
        const int at = pos + __popcll(km & lt);
        if (k && at < k_cap) idx_out[(size_t)seg * k_cap + at] = t;
        pos += __popcll(km);
    });
    if (tid == 0 && count_out != nullptr) count_out[seg] = total;
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
    const dim3 grid((unsigned)segs), block(kThreads);
    switch (R) {
#define KVE_TOPK_CASE(RR)                                                                                  \
    case RR:                                                                                               \
        hipLaunchKernelGGL(topk_kernel<RR>, grid, block, 0, st, score, roles, quota, B, Hkv, N, W, k_cap, \
                           idx_out, count_out);                                                            \
        break;
        KVE_TOPK_CASE(1)
        KVE_TOPK_CASE(2)
        KVE_TOPK_CASE(3)
        KVE_TOPK_CASE(4)
        KVE_TOPK_CASE(5)
        KVE_TOPK_CASE(6)
        KVE_TOPK_CASE(7)
        KVE_TOPK_CASE(8)
#undef KVE_TOPK_CASE
        default:
            return hipErrorInvalidValue;
    }
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
