// SnapKV windowed score with a single read of the keys (bf16).
//
// Paper: §2 (SnapKV: windowed mass over the last W queries, 1-D max-pool over
// the KV axis), §4 "SnapKV mechanism" and Algorithm 1 (windowed-mass step).
//
// The column sum of a key needs the log-sum-exp of every window row over all
// N keys.  The two-pass kernels therefore stream K twice; this kernel reads it
// once and keeps it on chip between the two uses:
//
//   * A work item is one vseg (a segment and a row group of 128 window rows)
//     and 256 of its keys.  A workgroup of four waves takes one item; each wave
//     loads its 64 keys straight into registers as matrix-core fragments (64
//     VGPRs) and the 128 query rows go to LDS, so the products need no key
//     traffic through LDS at all.
//   * Pass 1 (S^T = K Q^T, lane = query row) gives each row's log-sum-exp over
//     the item's keys.  The item publishes it and counts itself in at its
//     vseg; the last item of the vseg to arrive merges the partials and raises
//     the vseg's ready flag.  Every other item waits for the flag.
//   * Pass 2 (S = Q K^T, lane = key) takes the same key fragments: each wave
//     sums its 64 columns over all 128 rows with no cross-wave reduction, and
//     the raw column sums go to the same planes the pool step reads.
//
// Waiting cannot deadlock: items are handed out by an atomic ticket, so a
// vseg's items are taken by workgroups that are already running, and an item
// waits only after its own pass 1 is complete.  Every item of a vseg whose
// tickets are all taken therefore arrives.  A vseg's items are still waiting
// for untaken tickets only while fewer workgroups are resident than the vseg
// has items; the host uses this kernel only when the device holds at least
// twice that many.  Every wait is bounded all the same: after kSpinLimit polls
// the item stops waiting, sets the error word and writes NaN column sums, and
// every item that waits after that stops at once.
//
// Cross-workgroup data (partials, log-sum-exps, counters, flags) moves only
// through agent-scope atomic loads and stores, which are coherent across the
// L2 caches of all XCDs; an explicit vmcnt wait orders a workgroup's stores
// before its arrival.  No cache-wide fences are used.
//
// Logits are in log2 units (x = scale * log2(e) * <q, k>).  Within a lane the
// d dimension is split in two halves, so that each lane's fragments of one key
// are one contiguous run of the key row (D/2 elements) and the queries in LDS
// use the same split; the products sum over the same d values in another order.
#include "kve_device.h"
#include "kve_internal.h"
#include "kve_stream.h"

namespace kve {
namespace {

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * 64;
constexpr int kKeysPerWave = kSnap1ItemKeys / kWaves;  // 64: two 32-key blocks
constexpr int kRows = kSnapRowsPerGroup;               // 128: four 32-row blocks
constexpr unsigned kSpinLimit = 1u << 14;              // polls of a ready flag (about 10 ms)

static_assert(kKeysPerWave == 64, "two key blocks per wave");

using bf16 = __bf16;
using M = Mma<bf16>;

// Query rows sit in LDS at a pitch of ROW + 16 bytes: the 16-byte piece c of
// row r is in bank group r + c (mod the group count), so the consecutive rows
// that one LDS read cycle serves never share a group, and the piece of each
// k-step is an immediate offset from one per-lane address.
template <int D>
struct G1 {
    static constexpr int ROW = D * 2;       // bytes per query row
    static constexpr int PITCH = ROW + 16;  // bytes per query row in LDS
    static constexpr int NST = D / 16;      // k-steps of 16
    static constexpr int HALF = D / 2;      // d values per lane and key
    static constexpr int NC16 = ROW / 16;   // 16-byte pieces per row
};

struct Ctl {
    unsigned* ticket;
    unsigned* error;
    unsigned* count;  // per vseg
    unsigned* ready;  // per vseg
};

__device__ __forceinline__ Ctl ctl_of(unsigned* base, int n_vsegs) {
    return Ctl{base, base + 1, base + kSnap1CtlHead, base + kSnap1CtlHead + n_vsegs};
}

__device__ __forceinline__ void store_agent(float* p, float v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_agent(const float* p) {
    return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__global__ __launch_bounds__(256) void snap1_prep(unsigned* ctl, int words) {
    for (int i = blockIdx.x * 256 + threadIdx.x; i < words; i += gridDim.x * 256) ctl[i] = 0u;
}

template <int D>
__global__ __launch_bounds__(kThreads, 3) void snap1_score(const bf16* __restrict__ q, const bf16* __restrict__ k,
                                                           int N, int W, int rows, int rgroups, int nitems,
                                                           int n_vsegs, int segs, float sl2,
                                                           float* __restrict__ part, float* __restrict__ lse,
                                                           unsigned* __restrict__ ctl_base,
                                                           float* __restrict__ raw) {
    using Gd = G1<D>;
    __shared__ __align__(16) char qs[kRows * Gd::PITCH];  // the vseg's query rows
    __shared__ float2 spart[kWaves][kRows];             // per-wave (m, l) of each row
    __shared__ __align__(16) float sinit[kRows];        // -lse2 / sl2 of each row
    __shared__ __align__(16) int swin[kRows];           // window index of each row
    __shared__ int s_item, s_last, s_ok;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const Ctl ctl = ctl_of(ctl_base, n_vsegs);

    if (tid == 0) s_item = (int)__hip_atomic_fetch_add(ctl.ticket, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    const int item = s_item;
    const int vseg = item / nitems;
    const int range = item - vseg * nitems;
    const int seg = vseg / rgroups;
    const int rg = vseg - seg * rgroups;
    const int t_begin = range * kSnap1ItemKeys;
    const int t_end = min(N, t_begin + kSnap1ItemKeys);
    const int t0w = t_begin + wave * kKeysPerWave;  // first key of this wave
    const int P_rows = N - W;

    // Query rows of the vseg into LDS (zero for padding rows).
    {
        const char* qseg = reinterpret_cast<const char*>(q) + (size_t)seg * rows * Gd::ROW;
        constexpr int kPieces = kRows * Gd::NC16;
#pragma unroll
        for (int j = 0; j < kPieces / kThreads; ++j) {
            const int p = j * kThreads + tid;
            const int r = p / Gd::NC16, c = p % Gd::NC16;
            const int grow = rg * kRows + r;
            const u32x4 v = grow < rows ? ld16(qseg + (size_t)grow * Gd::ROW + c * 16) : zero16();
            st16(qs + r * Gd::PITCH + c * 16, v);
        }
        if (tid < kRows) swin[tid] = (rg * kRows + tid) % W;
    }
    // This wave's key fragments: block kb, k-step st = key t0w + 32 kb + lane % 32,
    // d values HALF * (lane / 32) + 8 st .. + 7.  Keys past the segment's end
    // read its last key (masked below).
    M::frag kf[2][Gd::NST];
    {
        const bf16* kseg = k + (size_t)seg * N * D;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            const int key = min(t0w + 32 * kb + (lane & 31), t_end - 1);
            const bf16* row = kseg + (size_t)key * D + (lane >> 5) * Gd::HALF;
#pragma unroll
            for (int st = 0; st < Gd::NST; ++st) kf[kb][st] = M::load(row, 8 * st);
        }
    }
    lds_barrier();  // query rows and window indices in LDS (the key loads stay in flight)
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int st = 0; st < Gd::NST; ++st) pin(kf[kb][st]);

    // query fragment (row block rb, k-step st) of this lane: row 32 rb + lane % 32,
    // d values HALF * (lane / 32) + 8 st .. + 7, at qlane + rb * 32 * PITCH + 16 st
    const char* qlane = qs + (lane & 31) * Gd::PITCH + (lane >> 5) * Gd::HALF * 2;
    const bool masked = t0w + kKeysPerWave > min(P_rows, t_end);  // wave-uniform

    // ---- pass 1: row statistics over this wave's 64 keys ----
    // S^T block of row block rb: element (kb, i) is key t0w + 32 kb + c_row(i, lane)
    // and row 32 rb + lane % 32; masked keys are -inf.
    auto products1 = [&](int rb, f32x16(&acc)[2]) {
        // masked keys start at -inf, which the products keep: no pass over the
        // results, whose registers the key fragments need
        if (masked) {
            // row rg * 128 + 32 rb + lane % 32 sees keys <= P_rows + row % W
            const int grow = rg * kRows + 32 * rb + (lane & 31);
            const int lim = grow < rows ? P_rows + swin[32 * rb + (lane & 31)] : -1;
            const int last = min(lim, t_end - 1) - (t0w + 4 * (lane >> 5));
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 16; ++i) acc[kb][i] = 32 * kb + 8 * (i >> 2) + (i & 3) > last ? -INFINITY : 0.0f;
        } else {
            acc[0] = f32x16{};
            acc[1] = f32x16{};
        }
#pragma unroll
        for (int st = 0; st < Gd::NST; ++st) {
            const M::frag qf = M::load(qlane + rb * 32 * Gd::PITCH + 16 * st, 0);
            acc[0] = M::mma(kf[0][st], qf, acc[0]);
            acc[1] = M::mma(kf[1][st], qf, acc[1]);
        }
    };
    // sum of exp2(sl2 * x - m) over the lane's 32 values, in place
    auto sum_from = [&](f32x16(&acc)[2], float m) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int i = 0; i < 16; ++i) acc[kb][i] = fast_exp2(fmaf(acc[kb][i], sl2, -m));
        float part[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
            part[e] = (acc[0][e] + acc[0][e + 4]) + (acc[0][e + 8] + acc[0][e + 12]) +
                      ((acc[1][e] + acc[1][e + 4]) + (acc[1][e + 8] + acc[1][e + 12]));
        return (part[0] + part[1]) + (part[2] + part[3]);
    };
    // Each row's (m, l) over the lane's 32 keys: the reference m is the largest
    // of four sampled logits, so the sum needs no full maximum.  When the sum
    // leaves [0, 2^64] (a logit more than 64 above the samples, or no finite
    // sample) the block is multiplied again and m is its exact maximum.
    float rm[4], rl[4];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
        f32x16 acc[2];
        products1(rb, acc);
        float m = fmaxf(fmaxf(acc[0][0], acc[0][8]), fmaxf(acc[1][0], acc[1][8])) * sl2;
        float l = sum_from(acc, m);
        if (!(l <= 0x1p64f)) {
            products1(rb, acc);
            float mx = -INFINITY;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 16; ++i) mx = fmaxf(mx, acc[kb][i]);
            m = mx * sl2;
            l = m == -INFINITY ? 0.0f : sum_from(acc, m);
        }
        rm[rb] = m;
        rl[rb] = l;
        // one row block at a time: reads hoisted from later blocks would hold
        // their fragments in registers next to the 64 of the keys
        __builtin_amdgcn_sched_barrier(0);
    }
    // the two lane halves hold the same rows and different keys
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
        lse2_merge(rm[rb], rl[rb], __shfl_xor(rm[rb], 32), __shfl_xor(rl[rb], 32));
        if (lane < 32) spart[wave][32 * rb + lane] = make_float2(rm[rb], rl[rb]);
    }
    __syncthreads();
    if (tid < kRows) {
        float m = -INFINITY, l = 0.0f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) lse2_merge(m, l, spart[w][tid].x, spart[w][tid].y);
        store_agent(&part[((size_t)vseg * nitems + range) * kRows + tid], (m != -INFINITY && l > 0.0f) ? m + log2f(l) : -INFINITY);
    }
    wait_vmcnt<0>();  // this wave's partials are performed before the arrival below
    __syncthreads();
    if (tid == 0) {
        const unsigned before = __hip_atomic_fetch_add(&ctl.count[vseg], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        s_last = before == (unsigned)(nitems - 1);
    }
    __syncthreads();

    // ---- the vseg's log-sum-exp of every row ----
    if (s_last) {
        // merge the partials of all items: thread (row, half) takes every other item
        const int r = tid & (kRows - 1), h = tid >> 7;
        float a = -INFINITY, b = 0.0f;
        const float* pr = part + (size_t)vseg * nitems * kRows + r;
        int c = h;
        for (; c + 14 < nitems; c += 16) {
            float v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = load_agent(pr + (size_t)(c + 2 * u) * kRows);
#pragma unroll
            for (int u = 0; u < 8; ++u) lse2_merge(a, b, v[u], v[u] == -INFINITY ? 0.0f : 1.0f);
        }
        for (; c < nitems; c += 2) {
            const float v = load_agent(pr + (size_t)c * kRows);
            lse2_merge(a, b, v, v == -INFINITY ? 0.0f : 1.0f);
        }
        spart[h][r] = make_float2(a, b);
        __syncthreads();
        if (tid < kRows) {
            lse2_merge(a, b, spart[1][tid].x, spart[1][tid].y);
            // rows past the window rows contribute nothing to the column sums
            const float v = (rg * kRows + tid < rows && b > 0.0f) ? a + log2f(b) : INFINITY;
            sinit[tid] = -v / sl2;
            store_agent(&lse[(size_t)vseg * kRows + tid], v);
        }
        wait_vmcnt<0>();
        __syncthreads();
        if (tid == 0) __hip_atomic_store(&ctl.ready[vseg], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    } else {
        if (tid == 0) {
            unsigned polls = 0;
            int ok = 1;
            while (__hip_atomic_load(&ctl.ready[vseg], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0u) {
                // give up after kSpinLimit polls, or at once when another item
                // has given up already (the grid then drains in one timeout)
                if (++polls > kSpinLimit ||
                    ((polls & 63u) == 0u &&
                     __hip_atomic_load(ctl.error, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u)) {
                    ok = 0;
                    __hip_atomic_store(ctl.error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    break;
                }
                __builtin_amdgcn_s_sleep(8);
            }
            s_ok = ok;  // not s_last: other waves may not have read it yet
        }
        __syncthreads();
        if (tid < kRows) sinit[tid] = s_ok ? -load_agent(&lse[(size_t)vseg * kRows + tid]) / sl2 : NAN;
    }
    __syncthreads();

    // ---- pass 2: column sums of this wave's 64 keys over the 128 rows ----
    // Element i of a block belongs to row 32 rb + c_row(i, lane) and the
    // lane's key; each starts at -lse2 / sl2 of its row, so that sl2 * acc is
    // x - lse2, and a masked one at -inf.
    auto start2 = [&](int rb, f32x16& acc) {
#pragma unroll
        for (int a = 0; a < 4; ++a) {
            const float4 v = *reinterpret_cast<const float4*>(&sinit[32 * rb + c_row(4 * a, lane)]);
            acc[4 * a] = v.x;
            acc[4 * a + 1] = v.y;
            acc[4 * a + 2] = v.z;
            acc[4 * a + 3] = v.w;
        }
    };
    auto lane_sum = [&](f32x16& acc) {
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[i] = fast_exp2(acc[i] * sl2);
        return ((acc[0] + acc[1]) + (acc[2] + acc[3]) + ((acc[4] + acc[5]) + (acc[6] + acc[7]))) +
               (((acc[8] + acc[9]) + (acc[10] + acc[11])) + ((acc[12] + acc[13]) + (acc[14] + acc[15])));
    };
    float cs[2] = {0.0f, 0.0f};
    if (!masked) {
        // both key blocks per query fragment read
#pragma unroll
        for (int rb = 0; rb < 4; ++rb) {
            f32x16 acc[2];
            start2(rb, acc[0]);
            acc[1] = acc[0];
#pragma unroll
            for (int st = 0; st < Gd::NST; ++st) {
                const M::frag qf = M::load(qlane + rb * 32 * Gd::PITCH + 16 * st, 0);
                acc[0] = M::mma(qf, kf[0][st], acc[0]);
                acc[1] = M::mma(qf, kf[1][st], acc[1]);
            }
            cs[0] += lane_sum(acc[0]);
            cs[1] += lane_sum(acc[1]);
            __builtin_amdgcn_sched_barrier(0);
        }
    } else {
        // keys in the causal window or past the end: one key block at a time,
        // so that the masks do not raise the register count of the kernel
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            const int t = t0w + 32 * kb + (lane & 31);  // key t is visible to window row w iff t - P_rows <= w
#pragma unroll
            for (int rb = 0; rb < 4; ++rb) {
                f32x16 acc;
                start2(rb, acc);
#pragma unroll
                for (int a = 0; a < 4; ++a) {
                    const int4 w4 = *reinterpret_cast<const int4*>(&swin[32 * rb + c_row(4 * a, lane)]);
                    const int wv[4] = {w4.x, w4.y, w4.z, w4.w};
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (!(t < t_end && t - P_rows <= wv[e])) acc[4 * a + e] = -INFINITY;
                }
#pragma unroll
                for (int st = 0; st < Gd::NST; ++st)
                    acc = M::mma(M::load(qlane + rb * 32 * Gd::PITCH + 16 * st, 0), kf[kb][st], acc);
                cs[kb] += lane_sum(acc);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    }
    float* out = raw + ((size_t)rg * segs + seg) * N;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
        const float v = cs[kb] + __shfl_xor(cs[kb], 32);  // the other 16 rows of each block
        const int t = t0w + 32 * kb + lane;
        if (lane < 32 && t < t_end) out[t] = v;
    }
}

template <int D>
int onepass_capacity(int device) {
    // resident workgroups of snap1_score on the device, cached per device
    static int cached[64] = {0};
    if (device < 0 || device >= 64) return 0;
    if (cached[device] == 0) {
        int per_cu = 0, cus = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(snap1_score<D>),
                                                         kThreads, 0) != hipSuccess)
            return 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess) return 0;
        cached[device] = per_cu * cus;
    }
    return cached[device];
}

template <int D>
hipError_t run_onepass(const void* q, const void* k, int L, int B, int Hq, int Hkv, int N, int W, float scale,
                       int pool_k, float* score, void* ws, hipStream_t st) {
    const SnapPlan p = snap_plan(L, B, Hq, Hkv, N, W, D);
    char* w = static_cast<char*>(ws);
    float* part = reinterpret_cast<float*>(w + p.off_part1);
    float* lse = reinterpret_cast<float*>(w + p.off_lse);
    float* raw = reinterpret_cast<float*>(w + p.off_raw);
    unsigned* ctl = reinterpret_cast<unsigned*>(w + p.off_ctl);
    const int words = kSnap1CtlHead + 2 * p.n_vsegs;
    hipLaunchKernelGGL(snap1_prep, dim3((unsigned)((words + 255) / 256 < 256 ? (words + 255) / 256 : 256)),
                       dim3(256), 0, st, ctl, words);
    const dim3 grid((unsigned)((size_t)p.n_vsegs * p.nitems1));
    hipLaunchKernelGGL((snap1_score<D>), grid, dim3(kThreads), 0, st, static_cast<const bf16*>(q),
                       static_cast<const bf16*>(k), N, W, p.rows, p.rgroups, p.nitems1, p.n_vsegs, p.segs,
                       scale * kLog2e, part, lse, ctl, raw);
    return launch_snap_pool(raw, p.planes, p.segs, N, W, pool_k, score, st);
}

}  // namespace

bool snapkv_onepass_fits(int dtype, int d, int nitems) {
    if (dtype != 0 || (d != 64 && d != 128)) return false;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return false;
    const int cap = d == 128 ? onepass_capacity<128>(dev) : onepass_capacity<64>(dev);
    return nitems >= 1 && 2 * nitems <= cap;
}

hipError_t launch_snapkv_onepass(const void* q, const void* k, int L, int B, int Hq, int Hkv, int N, int W,
                                 int d, float scale, int pool_k, float* score, void* ws, hipStream_t st) {
    if (d == 128) return run_onepass<128>(q, k, L, B, Hq, Hkv, N, W, scale, pool_k, score, ws, st);
    return run_onepass<64>(q, k, L, B, Hq, Hkv, N, W, scale, pool_k, score, ws, st);
}

}  // namespace kve
