// Per-role top-k selection (Algorithm 1, per-bucket top-k) with the window
// always kept, and the coalesced K/V compaction of the kept rows (§6: the
// dense cache of a compacting implementation).
//
// topk_select: one workgroup per (layer, sample, KV head) segment, of 4 waves,
// or of 16 when there are too few segments to fill the chip with 4-wave ones.
// Scores are mapped to order-preserving 32-bit keys (-0 -> +0, NaN lowest).
// Two sweeps read the segment's scores and labels:
//   1. Histogram sweep: the top 11 bits of every labelled candidate's key (sign,
//      exponent and two mantissa bits), one LDS histogram per bucket.  Per
//      bucket this gives the population, which decides whether the bucket is
//      kept whole, skipped or selected, and the top digit of the quota-th
//      largest key: the threshold's bin.
//   2. Staging sweep: each wave walks a contiguous share of the positions in
//      order and sets aside, in order, every position that is surely kept (the
//      window, whole buckets, keys above the threshold's bin) and every key
//      inside the bin (with its bucket and the low 21 bits of its key), in its
//      own part of the segment's workspace row (a position is staged at most
//      once, so a wave's part never overflows).
// Two more digit passes (11 and 10 bits) over the staged keys of the bins fix
// each bucket's threshold key and how many keys equal to it stay; each wave
// then walks its staged entries twice: it counts what it keeps (keys equal to
// a threshold are kept lowest position first, so the earlier waves' counts
// come first), then writes the kept positions in ascending order.
// In the sweeps a lane takes 16 consecutive positions per step: four 16-byte
// score loads and one 16-byte label load when the rows are 16-byte aligned,
// one load per position otherwise.  Bucket state is looked up per key in small
// LDS tables rather than picked from registers with a chain of selects.
#include <stdint.h>

#include "kve_device.h"
#include "kve_internal.h"

namespace kve {
namespace {

constexpr int kThreads = 256;        // top-k workgroup when segments fill the chip (and compaction)
constexpr int kWideThreads = 1024;   // top-k workgroup when there are few segments
constexpr int kWideBelow = 512;      // segments below which the wide workgroup is used
constexpr int kDigitBits = kRoleHistBits;  // the first digit is the fused score epilogue's histogram bin
constexpr int kDigits = 1 << kDigitBits;
constexpr int kLowBits = 32 - kDigitBits;  // key bits below the top digit
constexpr uint32_t kLowMask = (1u << kLowBits) - 1u;
constexpr int kSpan = 16;                  // consecutive positions per lane and step
constexpr int kWaveStep = kWave * kSpan;   // positions per wave step
constexpr int kBatch = 8;                  // staged entries per lane loaded before use
constexpr uint32_t kNoKey = 0xffffffffu;   // above every key (+inf maps to 0xff800000)
constexpr uint32_t kKept = 0xffffffffu;    // tag of a staged position that is surely kept

enum : int { kModeNone = 0, kModeSelect = 1, kModeAll = 2 };

template <int R, int NW>
struct TopkShared {
    uint32_t hist[R][kDigits];
    uint32_t pref[R];  // key bits fixed so far (bits lo .. 31)
    int lo[R];         // lowest fixed bit; 0 once the threshold is known
    int need[R];       // still to take among keys matching the prefix
    int mode[R];
    // staging: {lowest surely kept key, top digit of the threshold's bin} per
    // bucket; entry R (labels outside [0, R)) is never kept and never staged
    uint2 stage_cls[R + 1];
    int over;            // a fused-histogram tile of this segment overflowed its window
    int wave_eq[NW][R];  // staged keys equal to a threshold, per wave
    int wave_keep[NW];   // kept positions per wave
    int scan[NW][R < 4 ? R : 4];
};

// Exclusive prefix sums over a workgroup of NW waves of R values per thread (in
// thread order, each value on its own); every thread also gets the totals.
// `tmp` holds NW x R ints.
template <int R, int NW>
__device__ __forceinline__ void block_exclusive_scan(const int (&v)[R], int (&excl)[R], int (&total)[R],
                                                     int (*tmp)[R]) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int incl[R];
#pragma unroll
    for (int r = 0; r < R; ++r) incl[r] = v[r];
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int o = __shfl_up(incl[r], off);
            if (lane >= off) incl[r] += o;
        }
    }
    if (lane == kWave - 1) {
#pragma unroll
        for (int r = 0; r < R; ++r) tmp[wave][r] = incl[r];
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < R; ++r) {
        int before = 0, all = 0;
#pragma unroll
        for (int w = 0; w < NW; ++w) {
            const int t = tmp[w][r];
            if (w < wave) before += t;
            all += t;
        }
        excl[r] = before + incl[r] - v[r];
        total[r] = all;
    }
    __syncthreads();
}

// Exclusive prefix sum over the lanes of a wave of v in [0, 31] (lane order),
// and the wave's total: one ballot per bit.
__device__ __forceinline__ int wave_exclusive_scan(int v, int& total) {
    int excl = 0;
    total = 0;
#pragma unroll
    for (int bit = 0; bit < 5; ++bit) {
        const uint64_t m = __ballot((v >> bit) & 1);
        excl += (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u))
                << bit;
        total += __popcll(m) << bit;
    }
    return excl;
}

// Digit search of one pass for every bucket still selecting, in groups of up
// to four buckets (one scan per group, which bounds the registers the scan
// holds): thread tid holds kPerThread bins from the top going down per bucket;
// the scan gives the count of keys in all higher bins, and the thread whose
// bins reach a bucket's wanted rank fixes its digit.  In the first pass (quota
// given) the population decides whether a bucket is kept whole, skipped, or
// selected.  Every thread calls it.
constexpr int kScanGroup = 4;
template <int R, int NW>
__device__ __forceinline__ void find_digits(TopkShared<R, NW>& sh, const int32_t* quota) {
    constexpr int kPerThread = kDigits / (NW * kWave);
    constexpr int G = R < kScanGroup ? R : kScanGroup;
    const int tid = threadIdx.x;
    const int hi = kDigits - kPerThread * tid;  // bins [hi - kPerThread, hi)
#pragma unroll 1
    for (int r0 = 0; r0 < R; r0 += G) {
        // read before the scan's barriers: the threads that find the digits rewrite them
        bool act[G];
        int want[G], lo[G], mine[G];
#pragma unroll
        for (int g = 0; g < G; ++g) {
            const int r = r0 + g;
            act[g] = r < R && sh.mode[r] == kModeSelect && sh.lo[r] > 0;
            want[g] = act[g] ? sh.need[r] : 0;
            lo[g] = act[g] ? sh.lo[r] : 0;
            mine[g] = 0;
            if (act[g]) {
#pragma unroll
                for (int e = 1; e <= kPerThread; ++e) mine[g] += (int)sh.hist[r][hi - e];
            }
        }
        int above[G], total[G];
        block_exclusive_scan<G, NW>(mine, above, total, sh.scan);
#pragma unroll
        for (int g = 0; g < G; ++g) {
            const int r = r0 + g;
            if (!act[g]) continue;
            if (quota != nullptr) {
                const int q = max(quota[r], 0);
                if (q == 0 || q >= total[g]) {
                    if (tid == 0) sh.mode[r] = q == 0 ? kModeNone : kModeAll;
                    continue;
                }
                want[g] = q;
            }
            if (above[g] < want[g] && above[g] + mine[g] >= want[g]) {  // exactly one thread
                const int w = min(kDigitBits, lo[g]);
                int cum = above[g], dgt = hi - 1;
                for (; dgt > hi - kPerThread; --dgt) {
                    const int h = (int)sh.hist[r][dgt];
                    if (cum + h >= want[g]) break;
                    cum += h;
                }
                sh.pref[r] = (lo[g] < 32 ? sh.pref[r] << w : 0u) | (uint32_t)dgt;
                sh.need[r] = want[g] - cum;
                sh.lo[r] = lo[g] - w;
            }
        }
    }
    __syncthreads();
}

// Scores and labels of positions t0 .. t0 + 15 (label of t0 + 4 j + i: byte i
// of lab[j]).  VEC: t0 is a multiple of 16, the span lies inside the row and
// rows are 16-byte aligned; otherwise one load per position, the position
// clamped to [0, n).
template <bool VEC>
__device__ __forceinline__ void load_span(const float* sc, const int8_t* ro, int t0, int n, float (&s)[kSpan],
                                          uint32_t (&lab)[4]) {
    if constexpr (VEC) {
        const u32x4* sp = reinterpret_cast<const u32x4*>(sc + t0);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const u32x4 v = sp[j];
            s[4 * j] = __uint_as_float(v.x);
            s[4 * j + 1] = __uint_as_float(v.y);
            s[4 * j + 2] = __uint_as_float(v.z);
            s[4 * j + 3] = __uint_as_float(v.w);
        }
        const u32x4 l = *reinterpret_cast<const u32x4*>(ro + t0);
        lab[0] = l.x;
        lab[1] = l.y;
        lab[2] = l.z;
        lab[3] = l.w;
    } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            uint32_t w = 0u;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int t = min(t0 + 4 * j + i, n - 1);
                s[4 * j + i] = sc[t];
                w |= (uint32_t)(uint8_t)ro[t] << (8 * i);
            }
            lab[j] = w;
        }
    }
}

// bucket of the label of position t0 + e; R for labels outside [0, R)
template <int R>
__device__ __forceinline__ uint32_t bucket_of(const uint32_t (&lab)[4], int e) {
    return min((lab[e >> 2] >> (8 * (e & 3))) & 0xffu, (uint32_t)R);
}

template <int R, bool VEC, int NT>
__global__ __launch_bounds__(NT) void topk_kernel(const float* __restrict__ score, const int8_t* __restrict__ roles,
                                                  const int32_t* __restrict__ quota,
                                                  const uint32_t* __restrict__ hist_in, int B, int Hkv, int N,
                                                  int W, int k_cap, int32_t* __restrict__ idx_out,
                                                  int32_t* __restrict__ count_out, uint2* __restrict__ stage) {
    constexpr int NW = NT / kWave;
    constexpr int kGroupStep = NT * kSpan;  // positions per workgroup step
    __shared__ TopkShared<R, NW> sh;
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
    for (int e = tid; e < R * kDigits; e += NT) (&sh.hist[0][0])[e] = 0u;
    // 1. the first digit's counts: added up from the fused score epilogue's tile
    //    records when every tile fitted its window, otherwise counted in a sweep
    bool sweep = true;
    if (hist_in != nullptr) {
        const int tiles = (N + kRoleHistTile - 1) / kRoleHistTile;
        constexpr int kTw = kRoleHistHeader + R * kRoleHistWindow / 2;  // words per tile record
        const uint32_t* rec = hist_in + (size_t)seg * tiles * kTw;
        if (tid == 0) sh.over = 0;
        __syncthreads();
        for (int t = tid; t < tiles; t += NT)
            if (rec[(size_t)t * kTw + 1] != 0u) sh.over = 1;
        __syncthreads();  // also orders the zero fill before the adds
        sweep = sh.over != 0;  // uniform
        if (!sweep) {
            constexpr int kQ = R * kRoleHistWindow / 8;  // 16-byte words of count pairs per record
            for (int e = tid; e < tiles * kQ; e += NT) {
                const int t = e / kQ, q = e - t * kQ;
                const uint32_t* r0 = rec + (size_t)t * kTw;
                const uint32_t lo = r0[0];
                const u32x4 c = reinterpret_cast<const u32x4*>(r0 + kRoleHistHeader)[q];
                const int r = (4 * q) / (kRoleHistWindow / 2);
                const uint32_t bin0 = lo + 2u * (uint32_t)(4 * q - r * (kRoleHistWindow / 2));
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const uint32_t w = c[i], b = bin0 + 2u * i;
                    if ((w & 0xffffu) != 0u && b < (uint32_t)kDigits) atomicAdd(&sh.hist[r][b], w & 0xffffu);
                    if ((w >> 16) != 0u && b + 1u < (uint32_t)kDigits) atomicAdd(&sh.hist[r][b + 1], w >> 16);
                }
            }
        }
    }
    __syncthreads();
    if (sweep) {

    // 1. histogram sweep: the top digit of every labelled candidate's key; each
    //    step's span is in flight while the previous one is counted
    {
        float s[kSpan] = {}, sn[kSpan] = {};
        uint32_t lab[4] = {}, labn[4] = {};
        int t0 = kSpan * tid;
        if (t0 < P) load_span<VEC>(sc, ro, t0, N, s, lab);
        for (int base = 0; base < P; base += kGroupStep) {
            const int tn = t0 + kGroupStep;
            if (tn < P) load_span<VEC>(sc, ro, tn, N, sn, labn);
            if (t0 < P) {
                const int nv = min(kSpan, P - t0);
#pragma unroll
                for (int e = 0; e < kSpan; ++e) {
                    const uint32_t r = bucket_of<R>(lab, e);
                    if (e < nv && r < (uint32_t)R) atomicAdd(&sh.hist[r][score_key(s[e]) >> kLowBits], 1u);
                }
            }
#pragma unroll
            for (int e = 0; e < kSpan; ++e) s[e] = sn[e];
#pragma unroll
            for (int j = 0; j < 4; ++j) lab[j] = labn[j];
            t0 = tn;
        }
    }
    __syncthreads();
    }
    find_digits(sh, quota + (size_t)b * R);
    if (tid <= R) {
        uint2 c = make_uint2(kNoKey, kNoKey);
        if (tid < R && sh.mode[tid] == kModeAll) c.x = 0u;
        if (tid < R && sh.mode[tid] == kModeSelect) {
            // top digits are at most +inf's 0x7fc, so the shift does not overflow
            c.x = (sh.pref[tid] + 1u) << kLowBits;
            c.y = sh.pref[tid];
        }
        sh.stage_cls[tid] = c;
    }
    __syncthreads();

    // 2. staging sweep over this wave's run [w0, w1), in order
    const int run = (N + NW * kWaveStep - 1) / (NW * kWaveStep) * kWaveStep;
    const int w0 = min(N, wave * run), w1 = min(N, w0 + run);
    uint2* st = stage + (size_t)seg * N + w0;  // room for w1 - w0 entries
    int n_st = 0;
    {
        // each step's span is in flight while the previous one is staged; lanes
        // past the run load an in-bounds span and stage nothing
        float s[kSpan] = {}, sn[kSpan] = {};
        uint32_t lab[4] = {}, labn[4] = {};
        int t0 = w0 + kSpan * lane;
        if (w0 < w1) load_span<VEC>(sc, ro, VEC ? min(t0, N - kSpan) : t0, N, s, lab);
        for (int s0 = w0; s0 < w1; s0 += kWaveStep) {
            const int tn = t0 + kWaveStep;
            if (s0 + kWaveStep < w1) load_span<VEC>(sc, ro, VEC ? min(tn, N - kSpan) : tn, N, sn, labn);
            const int nv = max(0, min(kSpan, w1 - t0));
            uint32_t smask = 0u, tag[kSpan];
#pragma unroll
            for (int e = 0; e < kSpan; ++e) {
                const int t = t0 + e;
                const uint32_t key = score_key(s[e]);
                const uint32_t r = t < P ? bucket_of<R>(lab, e) : (uint32_t)R;
                const uint2 c = sh.stage_cls[r];
                const bool keep = t >= P || key >= c.x;
                const bool cand = (key >> kLowBits) == c.y;
                tag[e] = keep ? kKept : ((r << kLowBits) | (key & kLowMask));
                smask |= (e < nv && (keep || cand)) ? (1u << e) : 0u;
            }
            int tot;
            uint2* dst = st + n_st + wave_exclusive_scan(__popc(smask), tot);
#pragma unroll
            for (int e = 0; e < kSpan; ++e)
                if ((smask >> e) & 1u) *dst++ = make_uint2((uint32_t)(t0 + e), tag[e]);
            n_st += tot;
#pragma unroll
            for (int e = 0; e < kSpan; ++e) s[e] = sn[e];
#pragma unroll
            for (int j = 0; j < 4; ++j) lab[j] = labn[j];
            t0 = tn;
        }
    }
    __syncthreads();

    // the staged entries of this wave, kBatch per lane loaded before any is used;
    // visit(position, tag) for every entry in order, (0, kKept) with valid =
    // false past the end (every lane takes part in every step)
    auto sweep_staged = [&](auto&& visit) {
        for (int i0 = 0; i0 < n_st; i0 += kWave * kBatch) {
            uint2 ent[kBatch];
#pragma unroll
            for (int j = 0; j < kBatch; ++j) ent[j] = st[min(i0 + j * kWave + lane, n_st - 1)];
#pragma unroll
            for (int j = 0; j < kBatch; ++j) visit(ent[j].x, ent[j].y, i0 + j * kWave + lane < n_st);
        }
    };
    // full key of a staged key of a threshold bin
    auto bin_key = [&](uint32_t tg, uint32_t& r) {
        r = tg >> kLowBits;
        return (sh.stage_cls[r].y << kLowBits) | (tg & kLowMask);
    };

    // 3. the remaining digits (11 and 10 bits) over the staged keys of the bins
    for (int pass = 1; pass < 3; ++pass) {
        bool any = false;
#pragma unroll
        for (int r = 0; r < R; ++r) any |= sh.mode[r] == kModeSelect && sh.lo[r] > 0;
        if (!any) break;  // uniform: every thread reads the same LDS values
        for (int e = tid; e < R * kDigits; e += NT) (&sh.hist[0][0])[e] = 0u;
        __syncthreads();
        const int lo = 32 - kDigitBits * pass;  // the same for every selecting bucket
        const int w = min(kDigitBits, lo);
        sweep_staged([&](uint32_t, uint32_t tg, bool valid) {
            if (valid && tg != kKept) {
                uint32_t r;
                const uint32_t key = bin_key(tg, r);
                if ((key >> lo) == sh.pref[r]) atomicAdd(&sh.hist[r][(key >> (lo - w)) & ((1u << w) - 1u)], 1u);
            }
        });
        __syncthreads();
        find_digits(sh, static_cast<const int32_t*>(nullptr));
    }

    // 4. ordered output.  Class of a staged entry: 1 kept, 2 + r equal to bucket
    //    r's threshold, 0 dropped.
    int need[R];
#pragma unroll
    for (int r = 0; r < R; ++r) need[r] = sh.mode[r] == kModeSelect ? sh.need[r] : 0;
    auto classify = [&](uint32_t tg, bool valid) {
        if (!valid) return 0;
        if (tg == kKept) return 1;
        uint32_t r;
        const uint32_t key = bin_key(tg, r);
        const uint32_t th = sh.pref[r];
        return key > th ? 1 : (key == th ? 2 + (int)r : 0);
    };
    const uint64_t lt = (1ull << lane) - 1ull;
    int keep = 0, eq[R];
#pragma unroll
    for (int r = 0; r < R; ++r) eq[r] = 0;
    sweep_staged([&](uint32_t, uint32_t tg, bool valid) {
        const int c = classify(tg, valid);
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
    // equal keys are kept lowest position first: the earlier waves' come first
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
    for (int w = 0; w < NW; ++w) {
        if (w < wave) pos += sh.wave_keep[w];
        total += sh.wave_keep[w];
    }
    sweep_staged([&](uint32_t t, uint32_t tg, bool valid) {
        const int c = classify(tg, valid);
        bool k = c == 1;
        if (__ballot(c >= 2) != 0ull) {  // rare: keys equal to a threshold in this step
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const uint64_t m = __ballot(c == 2 + r);
                if (c == 2 + r) k = eq_seen[r] + (int)__popcll(m & lt) < need[r];
                eq_seen[r] += (int)__popcll(m);
            }
        }
        const uint64_t km = __ballot(k);
        const int at = pos + __popcll(km & lt);
        if (k && at < k_cap) idx_out[(size_t)seg * k_cap + at] = (int32_t)t;
        pos += __popcll(km);
    });
    if (tid == 0 && count_out != nullptr) count_out[seg] = total;
}

constexpr int kCompactRows = 64;

// One workgroup per (segment, 64 kept rows); a row is PARTS pieces of 16 bytes
// (8, 16 or 32), piece e of the block being part e % PARTS of row e / PARTS.
// Source rows are read through views (any row strides), the compacted rows
// are written dense.
// Every thread takes 64 PARTS / 256 pieces, in rounds of at most four: it
// issues the round's index loads, then its row loads, then its stores, so that
// a block waits for memory about twice per round instead of once per piece.
template <int PARTS>
__global__ __launch_bounds__(kThreads) void compact_kernel(RowView kv, RowView vv_, int B, int Hkv,
                                                           const int32_t* __restrict__ idx,
                                                           const int32_t* __restrict__ count, int N,
                                                           int k_cap, int nblk, char* __restrict__ k_out,
                                                           char* __restrict__ v_out) {
    constexpr int kRowBytes = PARTS * 16;
    constexpr int kItems = kCompactRows * PARTS / kThreads;
    constexpr int kRound = kItems < 4 ? kItems : 4;
    static_assert(kItems * kThreads == kCompactRows * PARTS && kItems % kRound == 0, "whole pieces per thread");
    const int blk = blockIdx.x % nblk;
    const int seg = blockIdx.x / nblk;
    const int cnt = min(count[seg], k_cap);
    const int m0 = blk * kCompactRows;
    if (m0 >= cnt) return;
    const int total = min(kCompactRows, cnt - m0) * PARTS;
    // segments are (layer, sample, KV head), KV head fastest
    const int lb = seg / Hkv;
    const long long so_k = (long long)(lb / B) * kv.s_layer + (long long)(lb % B) * kv.s_batch +
                           (long long)(seg % Hkv) * kv.s_head;
    const long long so_v = (long long)(lb / B) * vv_.s_layer + (long long)(lb % B) * vv_.s_batch +
                           (long long)(seg % Hkv) * vv_.s_head;
    const char* k = kv.base + so_k;
    const char* v = vv_.base != nullptr ? vv_.base + so_v : nullptr;
    const bool same_rows = vv_.s_token == kv.s_token;  // K and V rows equally spaced: one offset for both
    for (int i0 = 0; i0 < kItems; i0 += kRound) {
        if (i0 * kThreads >= total) break;  // uniform
        int t[kRound];
#pragma unroll
        for (int i = 0; i < kRound; ++i) {
            const int e = min((i0 + i) * kThreads + (int)threadIdx.x, total - 1);
            t[i] = idx[(size_t)seg * k_cap + m0 + e / PARTS];
        }
        u32x4 kr[kRound], vr[kRound];
#pragma unroll
        for (int i = 0; i < kRound; ++i) {
            const int e = min((i0 + i) * kThreads + (int)threadIdx.x, total - 1);
            const int tt = min(max(t[i], 0), N - 1);  // out-of-range indices are skipped below
            // token strides are below 2^25 bytes (checked by the caller): 32 x 32-bit products
            const unsigned piece = (unsigned)(e % PARTS) * 16u;
            const unsigned long long ko = (unsigned long long)(unsigned)tt * (unsigned)kv.s_token + piece;
            kr[i] = ld16(k + ko);
            if (v != nullptr)
                vr[i] = ld16(v + (same_rows ? ko : (unsigned long long)(unsigned)tt * (unsigned)vv_.s_token + piece));
        }
#pragma unroll
        for (int i = 0; i < kRound; ++i) {
            const int e = (i0 + i) * kThreads + (int)threadIdx.x;
            if (e < total && t[i] >= 0 && t[i] < N) {
                const size_t dst = ((size_t)seg * k_cap + m0 + e / PARTS) * kRowBytes + (size_t)(e % PARTS) * 16;
                st16(k_out + dst, kr[i]);
                if (v != nullptr) st16(v_out + dst, vr[i]);
            }
        }
    }
}

}  // namespace

hipError_t launch_topk(const float* score, const int8_t* roles, const int32_t* quota, const uint32_t* hist,
                       int L, int B, int Hkv, int N, int W, int R, int k_cap, int32_t* idx_out, int32_t* count_out,
                       void* ws, hipStream_t st) {
    const size_t segs = (size_t)L * B * Hkv;
    uint2* stage = static_cast<uint2*>(ws);
    // 16-byte span loads: every score row and label row starts 16-byte aligned
    const bool vec = N % kSpan == 0 && (reinterpret_cast<uintptr_t>(score) & 15u) == 0 &&
                     (reinterpret_cast<uintptr_t>(roles) & 15u) == 0;
    // few segments: sixteen waves per segment instead of four
    const bool wide = segs < (size_t)kWideBelow;
    const dim3 grid((unsigned)segs);
    switch (R) {
#define KVE_TOPK_LAUNCH(RR, V, NT)                                                                             \
    hipLaunchKernelGGL((topk_kernel<RR, V, NT>), grid, dim3(NT), 0, st, score, roles, quota, hist, B, Hkv, N, \
                       W, k_cap, idx_out, count_out, stage)
#define KVE_TOPK_CASE(RR)                                                                                      \
    case RR:                                                                                                   \
        if (wide) {                                                                                            \
            if (vec)                                                                                           \
                KVE_TOPK_LAUNCH(RR, true, kWideThreads);                                                       \
            else                                                                                               \
                KVE_TOPK_LAUNCH(RR, false, kWideThreads);                                                      \
        } else {                                                                                               \
            if (vec)                                                                                           \
                KVE_TOPK_LAUNCH(RR, true, kThreads);                                                           \
            else                                                                                               \
                KVE_TOPK_LAUNCH(RR, false, kThreads);                                                          \
        }                                                                                                      \
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
#undef KVE_TOPK_LAUNCH
        default:
            return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_compact(const RowView& k, const RowView& v, int elem_bytes, const int32_t* idx,
                          const int32_t* count, int L, int B, int Hkv, int N, int d, int k_cap,
                          void* k_out, void* v_out, hipStream_t st) {
    const size_t segs = (size_t)L * B * Hkv;
    const int nblk = (k_cap + kCompactRows - 1) / kCompactRows;
    if (nblk == 0 || segs == 0) return hipSuccess;
    const dim3 grid((unsigned)(segs * nblk));
    char* ko = static_cast<char*>(k_out);
    char* vo = static_cast<char*>(v_out);
    switch (d * elem_bytes / 16) {  // 16-byte pieces per row
        case 8:
            hipLaunchKernelGGL(compact_kernel<8>, grid, dim3(kThreads), 0, st, k, v, B, Hkv, idx, count, N, k_cap,
                               nblk, ko, vo);
            break;
        case 16:
            hipLaunchKernelGGL(compact_kernel<16>, grid, dim3(kThreads), 0, st, k, v, B, Hkv, idx, count, N, k_cap,
                               nblk, ko, vo);
            break;
        case 32:
            hipLaunchKernelGGL(compact_kernel<32>, grid, dim3(kThreads), 0, st, k, v, B, Hkv, idx, count, N, k_cap,
                               nblk, ko, vo);
            break;
        default:
            return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace kve
