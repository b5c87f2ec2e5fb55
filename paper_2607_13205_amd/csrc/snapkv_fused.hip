// SnapKV windowed score in one persistent launch that reads K from HBM once.
//
// Paper: §2 (SnapKV windowed mass), §4 "SnapKV mechanism", Algorithm 1
// (windowed-mass step).  The softmax of a window row needs its log-sum-exp over
// all N keys before any column sum can be formed, so every key is used twice:
// once for the row statistics and once for the column sums.  The second use
// reads the key chunk from LDS, not from HBM.
//
// Work items.  A virtual segment (vseg) is one (layer, sample, KV head, group
// of up to 128 window rows); its keys are cut into chunks of 64 keys.  The grid
// (two workgroups per CU) is launched cooperatively, so every workgroup is
// resident, with a size that is a multiple of the chunks per vseg; workgroup w
// takes items w, w+P, w+2P, ... so each round of P items holds whole vsegs.
//
// Software pipeline.  In iteration it a workgroup
//   - runs pass 1 on item it: S^T = K Q^T on the matrix cores; each lane holds
//     one query row and 16 keys per block, so the row maximum and the row sum
//     of exp2(x - max) reduce within the lane plus one cross-half shuffle; the
//     chunk's log-sum-exp of each row is published;
//   - merges its share of item it-1's vseg statistics: row r of a vseg is
//     merged by the workgroup whose chunk index is r mod the chunk count, into
//     lse2 = max + log2(sum), so the merge work is spread evenly;
//   - runs pass 2 on item it-2: S = Q K^T from the chunk still held in a
//     four-slot LDS ring (items it+1 .. it-2); each lane holds one key and 16
//     rows, so the column sum of exp2(x - lse2) is a lane sum plus one shuffle.
// Every value a wait depends on was published one full iteration earlier, so
// the waits normally find their counters complete.
//
// Wave roles.  A wave's vector-memory counter completes in issue order, so a
// wave that waits on a small load would also wait for any earlier chunk load.
// Waves 2 and 3 therefore stream the next key chunk straight into its LDS slot
// (16-byte direct-to-LDS loads, no register staging), and wave 0
// alone performs the traffic between workgroups: device-coherent loads and
// stores of statistics and lse2, and the completion flags.  Each workgroup
// raises its own flag word per (vseg, chunk) instead of adding to a shared
// counter, so no memory location is contended; a waiter reads all flags of a
// vseg in parallel across its 64 lanes.  Nothing needs a cache writeback or
// invalidate.  Each wait is bounded; a timeout sets the status word and later
// waits of that workgroup are skipped.
#include "kve_device.h"
#include "kve_internal.h"

namespace kve {
namespace {

constexpr int kThreads = 256;  // 4 waves, one 32-row block each
constexpr int kKeys = kFusedChunkKeys;  // keys per chunk (two 32-key blocks)
constexpr int kSlots = 4;      // LDS ring: items it+1, it, it-1, it-2
constexpr int kLoaders = 128;  // threads of waves 2 and 3
constexpr unsigned kSpinLimit = 1u << 20;  // ~50 ms of polling before giving up
constexpr int kMaxPairs = 8;   // chunk statistics a lane loads at once for its merge share

template <typename T, int D>
struct F {
    static constexpr int ES = (int)sizeof(T);
    static constexpr int ROW = D * ES;          // bytes per key row
    static constexpr int BUF = kKeys * ROW;     // bytes per chunk slot
    static constexpr int NB = kKeys / 32;       // 32-key blocks per chunk
    static constexpr int NC16 = ROW / 16;       // 16-byte pieces per row
    static constexpr int NSTEP = D / Mma<T>::KSTEP;
    static constexpr int LOADS = BUF / (kLoaders * 16);
};

template <typename T, int D>
using QFrag = typename Mma<T>::frag[F<T, D>::NSTEP];

// Byte offset of 16-byte piece c of key row r inside a slot (XOR swizzle: the
// 32 rows one matrix-core operand reads land on distinct bank groups).
template <typename T, int D>
__device__ __forceinline__ int swz(int r, int c) {
    return r * F<T, D>::ROW + ((c ^ (r & (F<T, D>::NC16 - 1))) << 4);
}

template <typename T, int D>
__device__ __forceinline__ typename Mma<T>::frag kfrag(const char* buf, int r, int k) {
    const int byte = k * F<T, D>::ES;
    return Mma<T>::load(buf + swz<T, D>(r, byte >> 4) + (byte & 15), 0);
}

struct Item {
    int vseg, seg, rg, chunk, t0;
};

__device__ __forceinline__ Item item_of(int item, int nchunks, int rgroups) {
    Item it;
    it.vseg = item / nchunks;
    it.chunk = item - it.vseg * nchunks;
    it.seg = it.vseg / rgroups;
    it.rg = it.vseg - it.seg * rgroups;
    it.t0 = it.chunk * kKeys;
    return it;
}

// Waves 2 and 3: stream a chunk into an LDS slot.  A direct-to-LDS load
// writes lane i's 16 bytes at (wave-uniform base) + 16 i, so each lane fetches
// the global piece that the swizzled layout keeps at that position.  Keys past
// N are not loaded (those slot bytes are only ever read under a mask).
template <typename T, int D>
__device__ __forceinline__ void stream_chunk(char* slot, const T* k, const Item& it, int N) {
    using S = F<T, D>;
    const char* base = reinterpret_cast<const char*>(k) + ((size_t)it.seg * N + it.t0) * S::ROW;
    const int lw = (threadIdx.x >> 6) - (kThreads - kLoaders) / 64;  // loader wave 0 or 1
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int j = 0; j < S::LOADS; ++j) {
        const int dst = (j * (kLoaders / 64) + lw) * 1024;  // wave-uniform byte offset
        const int o = dst + lane * 16;
        const int r = o / S::ROW;
        const int c = ((o - r * S::ROW) >> 4) ^ (r & (S::NC16 - 1));
        if (it.t0 + r < N)
            __builtin_amdgcn_global_load_lds(
                (const void __attribute__((address_space(1)))*)(base + r * S::ROW + c * 16),
                (void __attribute__((address_space(3)))*)(slot + dst), 16, 0, 0);
    }
}

template <typename T, int D>
__device__ __forceinline__ void load_q(QFrag<T, D>& qf, const T* q, int seg, int rows, int row) {
    using M = Mma<T>;
    const int lane = threadIdx.x & 63;
    const T* base = q + ((size_t)seg * rows + row) * D;
#pragma unroll
    for (int s = 0; s < F<T, D>::NSTEP; ++s)
        qf[s] = row < rows ? M::load(base, s * M::KSTEP + (lane >> 5) * M::KPL) : M::zero();
}

template <typename T, int D>
__device__ __forceinline__ void copy_q(QFrag<T, D>& dst, const QFrag<T, D>& src) {
#pragma unroll
    for (int s = 0; s < F<T, D>::NSTEP; ++s) dst[s] = src[s];
}

__device__ __forceinline__ float max3(float a, float b, float c) { return fmaxf(a, fmaxf(b, c)); }

// Device-coherent accesses for data shared between workgroups.
__device__ __forceinline__ void st_coh(float* p, float v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_coh(const float* p) {
    return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned ld_coh(const unsigned* p) {
    return __hip_atomic_load(const_cast<unsigned*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Every memory operation this wave issued has completed.
__device__ __forceinline__ void drain() { __builtin_amdgcn_s_waitcnt(0); }

__device__ __forceinline__ void st_coh(unsigned* p, unsigned v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Wave 0: poll until all n flags are set (bounded).
__device__ __forceinline__ void wait_flags(const unsigned* flags, int n, unsigned* err, bool& gave_up) {
    if (gave_up) return;
    const int lane = threadIdx.x & 63;
    unsigned spins = 0;
    while (true) {
        // issue every flag load of this lane before looking at any result
        bool mine = true;
        for (int j0 = 0; j0 < n; j0 += 64 * kMaxPairs) {
            unsigned v[kMaxPairs];
#pragma unroll
            for (int j = 0; j < kMaxPairs; ++j) {
                const int idx = j0 + lane + 64 * j;
                v[j] = idx < n ? ld_coh(flags + idx) : 1u;
            }
#pragma unroll
            for (int j = 0; j < kMaxPairs; ++j) mine &= v[j] != 0u;
        }
        if (__all(mine)) return;
        __builtin_amdgcn_s_sleep(1);
        if (++spins > kSpinLimit) {
            if (lane == 0) atomicOr(err, 1u);
            gave_up = true;
            return;
        }
    }
}

template <typename T, int D>
__global__ __launch_bounds__(kThreads, 2) void snap_stream(
    const T* __restrict__ q, const T* __restrict__ k, int N, int W, int rows, int rgroups, int nchunks,
    int n_items, float sl2, float* __restrict__ stats, float* __restrict__ lse,
    unsigned* __restrict__ arrive, unsigned* __restrict__ merged, unsigned* __restrict__ err, int segs,
    float* __restrict__ raw) {
    using M = Mma<T>;
    using S = F<T, D>;
    __shared__ __align__(16) char sbuf[kSlots][S::BUF];
    __shared__ float sstat[128];      // pass-1 chunk log-sum-exp (log2 units) per row
    __shared__ float slse[128];       // lse2 of the item in pass 2
    __shared__ float scol[4][kKeys];  // per-row-block column sums

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int P = gridDim.x;
    const int w = blockIdx.x;
    const int P_rows = N - W;
    const bool loader = tid >= kThreads - kLoaders;
    if (w >= n_items) return;
    const int n_it = (n_items - w + P - 1) / P;

    QFrag<T, D> q0, q1, q2;  // query fragments of items it, it-1, it-2
    bool gave_up = false;
    float lse_in[2] = {0.0f, 0.0f};

    Item cur = item_of(w, nchunks, rgroups);
    Item p1 = cur, p2 = cur;
    if (loader) {
        stream_chunk<T, D>(sbuf[0], k, cur, N);
        drain();
    }
    load_q<T, D>(q0, q, cur.seg, rows, cur.rg * 128 + wave * 32 + (lane & 31));

    for (int it = 0; it < n_it + 2; ++it) {
        const bool has0 = it < n_it;
        const bool has1 = it >= 1 && it - 1 < n_it;
        const bool has2 = it >= 2;
        const bool has_next = it + 1 < n_it;
        Item nxt = cur;
        if (has_next) nxt = item_of(w + (it + 1) * P, nchunks, rgroups);

        // ---- A: stream the next chunk (waves 2-3); fetch shared state (wave 0)
        if (loader && has_next) stream_chunk<T, D>(sbuf[(it + 1) % kSlots], k, nxt, N);
        if (wave == 0) {
            if (has1) wait_flags(arrive + (size_t)p1.vseg * nchunks, nchunks, err, gave_up);
            if (has2) wait_flags(merged + (size_t)p2.vseg * nchunks, nchunks, err, gave_up);
            __atomic_signal_fence(__ATOMIC_SEQ_CST);
            if (has2) {
                lse_in[0] = ld_coh(lse + (size_t)p2.vseg * 128 + lane);
                lse_in[1] = ld_coh(lse + (size_t)p2.vseg * 128 + 64 + lane);
            }
        }
        __syncthreads();

        // ---- C: pass 1 on item it (slot it % 3)
        if (has0) {
            const char* buf = sbuf[it % kSlots];
            const int qr = cur.rg * 128 + wave * 32 + (lane & 31);  // this lane's query row
            const int lim = qr < rows ? P_rows + (qr % W) : -1;
            float x[S::NB][16];
#pragma unroll
            for (int j = 0; j < S::NB; ++j) {
                f32x16 acc = {};
                const int r = 32 * j + (lane & 31);
#pragma unroll
                for (int s = 0; s < S::NSTEP; ++s)
                    acc = M::mma(kfrag<T, D>(buf, r, s * M::KSTEP + (lane >> 5) * M::KPL), q0[s], acc);
#pragma unroll
                for (int i = 0; i < 16; ++i) x[j][i] = acc[i];
            }
            if (cur.t0 + kKeys > P_rows) {  // keys past N or inside the causal window
#pragma unroll
                for (int j = 0; j < S::NB; ++j)
#pragma unroll
                    for (int i = 0; i < 16; ++i) {
                        const int t = cur.t0 + 32 * j + c_row(i, lane);
                        if (!(t < N && t <= lim)) x[j][i] = -INFINITY;
                    }
            }
            float m = -INFINITY;
#pragma unroll
            for (int j = 0; j < S::NB; ++j)
#pragma unroll
                for (int i = 0; i < 16; i += 2) m = max3(m, x[j][i], x[j][i + 1]);
            m = fmaxf(m, __shfl_xor(m, 32));
            float l = 0.0f;
            const float m2 = m * sl2;
            if (m != -INFINITY) {
#pragma unroll
                for (int j = 0; j < S::NB; ++j)
#pragma unroll
                    for (int i = 0; i < 16; ++i) l += fast_exp2(fmaf(x[j][i], sl2, -m2));
            }
            l += __shfl_xor(l, 32);
            if (lane < 32) sstat[wave * 32 + lane] = (m != -INFINITY && l > 0.0f) ? m2 + log2f(l) : -INFINITY;
        }
        __syncthreads();

        // ---- E: wave 0 merges its share of item it-1, publishes item it
        if (wave == 0) {
            if (has1) {
                for (int r = p1.chunk; r < 128; r += nchunks) {
                    float a = -INFINITY, b = 0.0f;
                    const float* sv = stats + (size_t)p1.vseg * nchunks * 128 + r;
                    for (int c0 = 0; c0 < nchunks; c0 += 64 * kMaxPairs) {
                        float mv[kMaxPairs];
#pragma unroll
                        for (int j = 0; j < kMaxPairs; ++j) {
                            const int c = c0 + lane + 64 * j;
                            mv[j] = c < nchunks ? ld_coh(sv + (size_t)c * 128) : -INFINITY;
                        }
#pragma unroll
                        for (int j = 0; j < kMaxPairs; ++j) lse2_merge(a, b, mv[j], mv[j] == -INFINITY ? 0.0f : 1.0f);
                    }
#pragma unroll
                    for (int off = 1; off < 64; off <<= 1) {
                        const float ao = __shfl_xor(a, off);
                        const float bo = __shfl_xor(b, off);
                        lse2_merge(a, b, ao, bo);
                    }
                    if (lane == 0) {
                        const int row = p1.rg * 128 + r;
                        // rows past the window rows contribute nothing to the column sums
                        st_coh(lse + (size_t)p1.vseg * 128 + r, (row < rows && b > 0.0f) ? a + log2f(b) : INFINITY);
                    }
                }
            }
            if (has0) {
                float* dst = stats + ((size_t)cur.vseg * nchunks + cur.chunk) * 128;
                st_coh(dst + lane, sstat[lane]);
                st_coh(dst + 64 + lane, sstat[64 + lane]);
            }
            if (has2) {
                slse[lane] = lse_in[0];
                slse[64 + lane] = lse_in[1];
            }
            drain();
            if (lane == 0) {
                if (has0) st_coh(arrive + (size_t)cur.vseg * nchunks + cur.chunk, 1u);
                if (has1) st_coh(merged + (size_t)p1.vseg * nchunks + p1.chunk, 1u);
            }
        }
        __syncthreads();

        // ---- G: pass 2 on item it-2 (slot (it-2) % 4 == (it+2) % 4)
        if (has2) {
            const char* buf = sbuf[(it + 2) % kSlots];
            const int row0 = p2.rg * 128 + wave * 32;
            float l2[16];
#pragma unroll
            for (int i = 0; i < 16; ++i) l2[i] = slse[wave * 32 + c_row(i, lane)];
            const bool full = p2.t0 + kKeys <= P_rows;
#pragma unroll
            for (int j = 0; j < S::NB; ++j) {
                f32x16 acc = {};
                const int r = 32 * j + (lane & 31);
#pragma unroll
                for (int s = 0; s < S::NSTEP; ++s)
                    acc = M::mma(q2[s], kfrag<T, D>(buf, r, s * M::KSTEP + (lane >> 5) * M::KPL), acc);
                float col = 0.0f;
                if (full) {
#pragma unroll
                    for (int i = 0; i < 16; ++i) col += fast_exp2(fmaf(acc[i], sl2, -l2[i]));
                } else {
                    const int t = p2.t0 + r;
#pragma unroll
                    for (int i = 0; i < 16; ++i) {
                        const int row = row0 + c_row(i, lane);
                        const bool ok = t < N && row < rows && t <= P_rows + (row % W);
                        col += ok ? fast_exp2(fmaf(acc[i], sl2, -l2[i])) : 0.0f;
                    }
                }
                col += __shfl_xor(col, 32);
                if (lane < 32) scol[wave][32 * j + lane] = col;
            }
        }
        __syncthreads();

        // ---- I: write the column sums; refill the freed slot; rotate
        if (has2 && tid < kKeys) {
            const int t = p2.t0 + tid;
            if (t < N)
                raw[((size_t)p2.rg * segs + p2.seg) * N + t] =
                    (scol[0][tid] + scol[1][tid]) + (scol[2][tid] + scol[3][tid]);
        }
        if (loader && has_next) drain();  // chunk it+1 has landed in its slot
        copy_q<T, D>(q2, q1);
        copy_q<T, D>(q1, q0);
        p2 = p1;
        p1 = cur;
        if (has_next) {
            cur = nxt;
            load_q<T, D>(q0, q, cur.seg, rows, cur.rg * 128 + wave * 32 + (lane & 31));
        }
    }
}

__global__ void snap_stream_reset(unsigned* __restrict__ arrive, unsigned* __restrict__ merged,
                                  unsigned* __restrict__ err, size_t n) {
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += stride) {
        arrive[i] = 0u;
        merged[i] = 0u;
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) err[0] = 0u;
}

template <typename T, int D>
int resident_blocks() {
    static int cached = -1;
    if (cached < 0) {
        int dev = 0, cus = 0, per_cu = 0;
        if (hipGetDevice(&dev) != hipSuccess) return 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, snap_stream<T, D>, kThreads, 0) != hipSuccess)
            return 0;
        cached = cus * per_cu;
    }
    return cached;
}

template <typename T, int D>
hipError_t run_fused(const void* q, const void* k, int L, int B, int Hq, int Hkv, int N, int W,
                     float scale, float* raw, void* ws, hipStream_t st, bool* used) {
    *used = false;
    const SnapPlan p = snap_plan(L, B, Hq, Hkv, N, W, D);
    const int nchunks = (N + kKeys - 1) / kKeys;
    const long long n_items = (long long)p.n_vsegs * nchunks;
    const int cap = resident_blocks<T, D>();
    if (cap <= 0 || nchunks > cap || nchunks > p.fchunks_max || n_items > 0x7fffffffLL) return hipSuccess;
    int P = cap / nchunks * nchunks;
    if (P > n_items) P = (int)n_items;
    char* w = static_cast<char*>(ws);
    unsigned* errw = reinterpret_cast<unsigned*>(w + p.off_err);
    unsigned* arrive = reinterpret_cast<unsigned*>(w + p.off_arrive);
    unsigned* merged = reinterpret_cast<unsigned*>(w + p.off_ready);
    float* stats = reinterpret_cast<float*>(w + p.off_fstats);
    float* lse = reinterpret_cast<float*>(w + p.off_flse);
    const size_t n_flags = (size_t)p.n_vsegs * nchunks;
    const unsigned reset_blocks = (unsigned)((n_flags + 255) / 256 < 4096 ? (n_flags + 255) / 256 : 4096);
    hipLaunchKernelGGL(snap_stream_reset, dim3(reset_blocks), dim3(256), 0, st, arrive, merged, errw, n_flags);
    const T* qt = static_cast<const T*>(q);
    const T* kt = static_cast<const T*>(k);
    int Nn = N, Wn = W, rows = p.rows, rg = p.rgroups, nch = nchunks, nit = (int)n_items, segs = p.segs;
    float sl2 = scale * kLog2e;
    void* args[] = {(void*)&qt,    (void*)&kt,     (void*)&Nn,   (void*)&Wn,    (void*)&rows, (void*)&rg,
                    (void*)&nch,   (void*)&nit,    (void*)&sl2,  (void*)&stats, (void*)&lse,  (void*)&arrive,
                    (void*)&merged, (void*)&errw,  (void*)&segs, (void*)&raw};
    const hipError_t e = hipLaunchCooperativeKernel(reinterpret_cast<const void*>(snap_stream<T, D>), dim3(P),
                                                    dim3(kThreads), args, 0, st);
    if (e == hipErrorCooperativeLaunchTooLarge) {
        (void)hipGetLastError();  // the two-pass kernels take over
        return hipSuccess;
    }
    if (e == hipSuccess) *used = true;
    return e;
}

}  // namespace

hipError_t launch_snapkv_fused(const void* q, const void* k, int dtype, int L, int B, int Hq, int Hkv, int N,
                               int W, int d, float scale, float* raw, void* ws, hipStream_t st, bool* used) {
    if (dtype == 0) {
        if (d == 128) return run_fused<__bf16, 128>(q, k, L, B, Hq, Hkv, N, W, scale, raw, ws, st, used);
        return run_fused<__bf16, 64>(q, k, L, B, Hq, Hkv, N, W, scale, raw, ws, st, used);
    }
    if (d == 128) return run_fused<float, 128>(q, k, L, B, Hq, Hkv, N, W, scale, raw, ws, st, used);
    return run_fused<float, 64>(q, k, L, B, Hq, Hkv, N, W, scale, raw, ws, st, used);
}

}  // namespace kve
