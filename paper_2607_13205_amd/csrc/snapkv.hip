// SnapKV windowed score with fused GQA sum and prefix max-pool: streaming
// two-pass kernels.
//
// Paper: §2 (SnapKV: windowed mass over the last W queries, 1-D max-pool over
// the KV axis), §4 "SnapKV mechanism" (pool kernel 7) and Algorithm 1
// (windowed-mass and pooling steps).
//
// A segment is one (layer, sample, KV head); its rows are the G*W window
// queries of the group (head-major), taken in row groups of 128, or of 256 for
// bf16 windows of more than 128 rows (a virtual segment, vseg, is one segment
// and one row group).  A workgroup of four waves owns a vseg and a contiguous
// range of its keys; each wave owns one 32-row block, or two, whose query
// fragments stay in registers.  Keys stream through an LDS
// ring in chunks of 64 with direct-to-LDS loads issued one to three chunks
// ahead, so every wave keeps HBM requests in flight while it multiplies on the
// matrix cores (bf16 32x32x16, fp32 32x32x2).  No workgroup waits on another
// one; two to four workgroups share a compute unit, so that one's matrix-core
// work overlaps another's exponentials.
//
//   pass 1   snap_pass1    S^T = K Q^T: each lane holds one row and 16 keys per
//                          32-key block, so the running row sum of
//                          exp2(x - ref) stays in the lane; one log-sum-exp per
//                          (vseg, range, row) is written.
//   combine  snap_combine  per row: lse2 over the ranges (+inf for padding rows).
//   pass 2   snap_pass2    S = Q K^T: each lane holds one key and 16 rows per
//                          block, so the column sum of exp2(x - lse2) is a lane
//                          sum plus one shuffle; the four row blocks (waves)
//                          add through LDS and each chunk's 64 sums go out.
//   pool     snap_pool     adds the row groups and max-pools the prefix.
//
// Logits are kept in log2 units (x = scale * log2(e) * <q, k>) so that every
// exponential is a single v_exp_f32.
#include <cstring>
#include <mutex>

#include "kve_device.h"
#include "kve_internal.h"
#include "kve_snap_plan.h"
#include "kve_stream.h"

// Workspace of the allocation-free entry point: a static device array, one
// copy per GPU the library runs on.  In host code its name is not a device
// address; kernels only ever receive the address snapkv_scratch() returns.
static __device__ __align__(256) char scratch[kve::kSnapScratchBytes];

namespace kve {
namespace {

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * 64;
constexpr int kKeys = kSnapChunkKeys;  // keys per chunk
// keys per pool workgroup: 2048 when it only pools (twice the workgroups of
// 4096-key tiles hide more of the plane reads: measured 97 -> 58 us on a 32k
// stack), the role-histogram tile when it also counts (its records then stay
// as few as the top-k reads)
constexpr int kPoolTile = 2048;
constexpr int kMaxPoolHalf = 127;

// LDS ring depth and workgroups per compute unit of each pass.  bf16: both
// passes keep one chunk in flight at four workgroups per CU (with non-temporal
// chunk loads and conflict-free fragment reads, the fourth workgroup hides more
// than a second chunk ahead: measured 1-2% faster than two chunks at three);
// the extra workgroup also overlaps more of one wave's exponentials with
// another's products.
// fp32 fragments need twice the registers: two workgroups, three chunks ahead
// (one workgroup at d = 128, whose 32 KB chunks fill LDS with the ring).
template <typename T>
struct Tune {
    static constexpr int kRing1 = 4, kOcc1 = 2, kRing2 = 4, kOcc2 = 2;
};
template <>
struct Tune<__bf16> {
    static constexpr int kRing1 = 2, kOcc1 = 4, kRing2 = 2, kOcc2 = 4;
};
// two 32-row sets per wave (bf16, windows of more than 128 rows): twice the
// query fragments and accumulators, two chunks ahead, three workgroups per CU
// (168 registers): pass 1 takes its exponentials in place of the logits, pass
// 2 reads its start values from LDS into the accumulators at every chunk
// (4-5% faster per pass than two workgroups on the 32-layer, N = 131072,
// W = 64 workload)
template <typename T, int RS>
struct TuneRS : Tune<T> {};
template <typename T>
struct TuneRS<T, 2> {
    static constexpr int kRing1 = 3, kOcc1 = 3, kRing2 = 3, kOcc2 = 3;
};

// Each pass reads every key row once: non-temporal chunk loads (measured 3-4%
// faster per pass than cached ones on the 32-layer, N = 32768 workload).
template <typename T, int D, int RING>
struct Geo {
    using C = KChunk<T, D, kKeys>;
    using Rd = ChunkReader<T, D, kKeys>;
    using Ring = ChunkRing<T, D, kKeys, kWaves, RING, true>;
};

struct Span {
    int vseg, seg, rg, range, t_begin, t_end, nch;
};

// Fused role epilogue of the pool step: one tile record per (segment, pool
// tile) of the role histograms (layout in kve_snap_plan.h).  roles == nullptr:
// no histogram.
struct RoleHist {
    const int8_t* roles;  // [B, N] bucket labels; labels outside [0, R) are not counted
    uint32_t* hist;       // [segs, tiles, role_hist_tile_words(R)]
    int R, B, Hkv;
    uint32_t lo;          // first bin of every tile's window
};

__device__ __forceinline__ Span span_of(int nranges, int rgroups, int range_keys, int N) {
    Span s;
    s.vseg = blockIdx.x / nranges;
    s.range = blockIdx.x - s.vseg * nranges;
    s.seg = s.vseg / rgroups;
    s.rg = s.vseg - s.seg * rgroups;
    s.t_begin = s.range * range_keys;
    s.t_end = min(N, s.t_begin + range_keys);
    s.nch = (s.t_end - s.t_begin + kKeys - 1) / kKeys;
    return s;
}

// Query fragments of this wave's 32-row block (zero for padding rows).
template <typename T, int D>
using QRows = typename Mma<T>::frag[KChunk<T, D, kKeys>::NSTEP];

// Start of segment seg's rows in a view whose head dimension has `heads`
// heads per segment (1 for keys, G for the queries of a KV group): segments
// are (layer, sample, KV head), KV head fastest.
__device__ __forceinline__ const char* seg_rows(const RowView& v, int seg, int B, int Hkv, int heads) {
    const int j = seg % Hkv;
    const int lb = seg / Hkv;
    return v.base + (long long)(lb / B) * v.s_layer + (long long)(lb % B) * v.s_batch +
           (long long)j * heads * v.s_head;
}

// row: the segment's window row g W + i (query head g of the group, window
// position i); qseg: the group's first query head (seg_rows with heads G)
template <typename T, int D>
__device__ __forceinline__ void load_q(QRows<T, D>& qf, const char* qseg, const RowView& qv, int rows, int W,
                                       int row, int lane) {
    using M = Mma<T>;
    const char* base = qseg + (long long)(row / W) * qv.s_head + (long long)(row % W) * qv.s_token;
#pragma unroll
    for (int st = 0; st < KChunk<T, D, kKeys>::NSTEP; ++st) {
        qf[st] = row < rows ? M::load(base, st * M::KSTEP + (lane >> 5) * M::KPL) : M::zero();
        pin(qf[st]);
    }
}

// Chunks of a key range of one segment: chunk c starts at key t_begin + 64 c;
// key rows are `stride` bytes apart.
template <typename T, int D>
struct KeyChunks {
    const char* kseg;
    long long stride;
    int t_begin, t_end;
    __device__ __forceinline__ void operator()(int c, const char** rows, int* valid) const {
        const int t0 = t_begin + c * kKeys;
        *rows = kseg + (long long)t0 * stride;
        *valid = t_end - t0;
    }
};

template <typename T, int D, int RS>
__global__ __launch_bounds__(kThreads, (sizeof(T) == 4 && D == 128 ? 1 : TuneRS<T, RS>::kOcc1)) void snap_pass1(
    RowView qv, RowView kv, int B, int Hkv, int N, int W, int rows, int rgroups, int nranges, int range_keys,
    float sl2, float* __restrict__ stats) {
    constexpr int kRing = TuneRS<T, RS>::kRing1;
    constexpr int kRpg = RS * kSnapRowsPerGroup;
    using G = Geo<T, D, kRing>;
    __shared__ __align__(16) char ring[kRing * G::C::BYTES];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const Span sp = span_of(nranges, rgroups, range_keys, N);
    const int P_rows = N - W;

    // wave w holds rows 32 RS w .. 32 RS (w + 1) - 1 of the row group, in RS sets of 32
    const char* qseg = seg_rows(qv, sp.seg, B, Hkv, rows / W);
    QRows<T, D> qf[RS];
    auto qrow = [&](int rs) { return sp.rg * kRpg + (wave * RS + rs) * 32 + (lane & 31); };  // this lane's query row
#pragma unroll
    for (int rs = 0; rs < RS; ++rs) load_q<T, D>(qf[rs], qseg, qv, rows, W, qrow(rs), lane);
    typename G::Rd rd;
    rd.init(lane, 0);
    typename G::Ring ring_io;
    ring_io.open(sp.nch, wave, lane, (unsigned)kv.s_token);
    const KeyChunks<T, D> src{seg_rows(kv, sp.seg, B, Hkv, 1), kv.s_token, sp.t_begin, sp.t_end};
    ring_io.prologue(ring, src);

    // the logits of chunk s (ring slot u), masked past the range end and
    // inside the causal window
    auto logits = [&](f32x16 (&acc)[RS][2], int s, int u) {
        chunk_mma_sets<T, D, kKeys, true, RS>(acc, rd, ring + u * G::C::BYTES, qf, nullptr);
        if (sp.t_begin + (s + 1) * kKeys > P_rows) {
#pragma unroll
            for (int rs = 0; rs < RS; ++rs) {
                const int qr = qrow(rs);
                const int lim = qr < rows ? P_rows + qr % W : -1;  // last key the row sees
                // key of element (kb, i) = base + 32 kb + 8 (i / 4) + i % 4; a
                // key past `last` gets -inf added (the sign of last - key
                // picks -inf or +0), which keeps the per-element tests out of
                // the scalar registers a compare-and-select would hold them in
                const int last = min(lim, sp.t_end - 1) - (sp.t_begin + s * kKeys + 4 * (lane >> 5));
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int i = 0; i < 16; ++i)
                        acc[rs][kb][i] += __int_as_float(((last - (32 * kb + 8 * (i >> 2) + (i & 3))) >> 31) &
                                                         (int)0xff800000u);
            }
        }
    };
    RowSum rsum[RS];
    for (int s0 = 0; s0 < sp.nch; s0 += kRing) {
#pragma unroll
        for (int u = 0; u < kRing; ++u) {
            const int s = s0 + u;
            if (s >= sp.nch) break;
            ring_io.advance(ring, s, u, src);
            f32x16 acc[RS][2];
            logits(acc, s, u);
            float ln[RS];
            if (!row_sums_try<RS>(rsum, acc, sl2, ln)) {
                // a sum left [0, 2^64]: the exponentials replaced the logits,
                // and the chunk stays in its slot until the next barrier
                logits(acc, s, u);
                row_sums_fix<RS>(rsum, acc, sl2, ln);
            }
        }
    }
#pragma unroll
    for (int rs = 0; rs < RS; ++rs) {
        // the two lane halves hold the same row and different keys
        lse2_merge(rsum[rs].m, rsum[rs].l, __shfl_xor(rsum[rs].m, 32), __shfl_xor(rsum[rs].l, 32));
        if (lane < 32)
            stats[((size_t)sp.vseg * nranges + sp.range) * kRpg + (wave * RS + rs) * 32 + lane] = rsum[rs].lse2();
    }
}

// Four threads per row of a row group (thread 4 r + s, rpg = blockDim.x / 4
// rows): thread s merges every fourth range from range s, 32 ranges' values
// loaded before any is merged, then the four partial sums of a row merge by
// shuffles.
constexpr int kCombineSplit = 4;
__global__ __launch_bounds__(2 * kSnapRowsPerGroup * kCombineSplit) void snap_combine(
    const float* __restrict__ stats, int nranges, int rows, int rgroups, float* __restrict__ lse) {
    const int vseg = blockIdx.x, rpg = blockDim.x / kCombineSplit;
    const int r = threadIdx.x / kCombineSplit, sub = threadIdx.x % kCombineSplit;
    const int row = (vseg % rgroups) * rpg + r;
    float a = -INFINITY, b = 0.0f;
    for (int c0 = sub; c0 < nranges; c0 += 32 * kCombineSplit) {
        float v[32];
#pragma unroll
        for (int j = 0; j < 32; ++j)
            v[j] = stats[((size_t)vseg * nranges + min(c0 + j * kCombineSplit, nranges - 1)) * rpg + r];
#pragma unroll
        for (int j = 0; j < 32; ++j)
            if (c0 + j * kCombineSplit < nranges) lse2_merge(a, b, v[j], v[j] == -INFINITY ? 0.0f : 1.0f);
    }
#pragma unroll
    for (int m = 1; m < kCombineSplit; m <<= 1) {
        const float ao = __shfl_xor(a, m), bo = __shfl_xor(b, m);
        lse2_merge(a, b, ao, bo);
    }
    // rows past the window rows contribute nothing to the column sums
    if (sub == 0) lse[(size_t)vseg * rpg + r] = (row < rows && b > 0.0f) ? a + log2f(b) : INFINITY;
}

// Row statistics supplied by the caller (the natural-log log-sum-exp of each
// window row, [segments, G, W] as a prefill attention kernel returns it per
// query row), turned into the combine step's output: log2 units, rows of the
// vseg layout, +inf for padding rows.
// one thread per row of a row group (rpg = blockDim.x rows)
__global__ __launch_bounds__(2 * kSnapRowsPerGroup) void snap_import_lse(const float* __restrict__ lse_win,
                                                                         int rows, int rgroups,
                                                                         float* __restrict__ lse) {
    const int vseg = blockIdx.x, r = threadIdx.x, rpg = blockDim.x;
    const int seg = vseg / rgroups;
    const int row = (vseg - seg * rgroups) * rpg + r;  // head-major: g * W + i
    lse[(size_t)vseg * rpg + r] = row < rows ? lse_win[(size_t)seg * rows + row] * kLog2e : INFINITY;
}

template <typename T, int D, int RS>
__global__ __launch_bounds__(kThreads, (sizeof(T) == 4 && D == 128 ? 1 : TuneRS<T, RS>::kOcc2)) void snap_pass2(
    RowView qv, RowView kv, int B, int Hkv, int N, int W, int rows, int rgroups, int nranges, int range_keys,
    float sl2, const float* __restrict__ lse, int segs, float* __restrict__ raw) {
    constexpr int kRing = TuneRS<T, RS>::kRing2;
    constexpr int kRpg = RS * kSnapRowsPerGroup;
    using G = Geo<T, D, kRing>;
    __shared__ __align__(16) char ring[kRing * G::C::BYTES];
    __shared__ __align__(16) float scol[2][kKeys][kWaves];  // column sums per key and wave, two chunks
    __shared__ __align__(16) float sinit[kRpg];  // -lse / sl2 of each row
    __shared__ __align__(16) int swin[kRpg];     // window index (row % W) of each row
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const Span sp = span_of(nranges, rgroups, range_keys, N);
    const int P_rows = N - W;

    // The products start from -lse / sl2 of their row, so that sl2 * acc is
    // x - lse2 directly (the accumulator is float32: the offset costs no
    // precision that matters); padding rows (lse = +inf) start at -inf and add
    // exactly 0.  The window index of each row stays in LDS for the masked
    // path: as registers the 32 loop-invariant bounds would stay live across
    // the whole loop.
    for (int r = threadIdx.x; r < kRpg; r += kThreads) {
        sinit[r] = -lse[(size_t)sp.vseg * kRpg + r] / sl2;
        swin[r] = (sp.rg * kRpg + r) % W;
    }
    // wave w holds rows 32 RS w .. 32 RS (w + 1) - 1 of the row group, in RS sets of 32
    const char* qseg = seg_rows(qv, sp.seg, B, Hkv, rows / W);
    QRows<T, D> qf[RS];
#pragma unroll
    for (int rs = 0; rs < RS; ++rs)
        load_q<T, D>(qf[rs], qseg, qv, rows, W, sp.rg * kRpg + (wave * RS + rs) * 32 + (lane & 31), lane);
    __syncthreads();  // sinit, swin written (nothing streams yet)
    // start values of this lane's 16 rows of each set, the same for every
    // chunk: held in registers with one set per wave; with two sets read from
    // LDS into the accumulators at every chunk instead (32 registers fewer,
    // which lets three workgroups share a CU; all 32 lanes of a half-wave read
    // the same 16 bytes, so the reads are broadcasts)
    constexpr bool kInitLds = RS == 2;
    f32x16 c_init[RS];
    if constexpr (!kInitLds) {
#pragma unroll
        for (int rs = 0; rs < RS; ++rs) {
#pragma unroll
            for (int a = 0; a < 4; ++a) {
                const float4 v = *reinterpret_cast<const float4*>(&sinit[(wave * RS + rs) * 32 + c_row(4 * a, lane)]);
                c_init[rs][4 * a] = v.x;
                c_init[rs][4 * a + 1] = v.y;
                c_init[rs][4 * a + 2] = v.z;
                c_init[rs][4 * a + 3] = v.w;
            }
            pin(c_init[rs]);
        }
    }
    typename G::Rd rd;
    rd.init(lane, 0);
    typename G::Ring ring_io;
    ring_io.open(sp.nch, wave, lane, (unsigned)kv.s_token);
    const KeyChunks<T, D> src{seg_rows(kv, sp.seg, B, Hkv, 1), kv.s_token, sp.t_begin, sp.t_end};
    ring_io.prologue(ring, src);
    float* out = raw + ((size_t)sp.rg * segs + sp.seg) * N;

    // add the four waves' column sums of chunk s (every wave has written them):
    // the waves take the chunks in turn, lane l adding the four sums of key l
    // (one 16-byte LDS read) and the wave writing all 64 as one 256-byte store
    auto reduce = [&](int s) {
        if (wave == (s & (kWaves - 1))) {
            const int t = sp.t_begin + s * kKeys + lane;
            const float4 c = *reinterpret_cast<const float4*>(&scol[s & 1][lane][0]);
            if (t < sp.t_end) out[t] = (c.x + c.y) + (c.z + c.w);
        }
    };
    for (int s0 = 0; s0 < sp.nch; s0 += kRing) {
#pragma unroll
        for (int u = 0; u < kRing; ++u) {
            const int s = s0 + u;
            if (s >= sp.nch) break;
            f32x16 acc[RS][2];
            if constexpr (kInitLds) {  // before the wait: the reads' latency hides behind it
#pragma unroll
                for (int rs = 0; rs < RS; ++rs)
#pragma unroll
                    for (int b = 0; b < 2; ++b)
#pragma unroll
                        for (int a = 0; a < 4; ++a) {
                            const float4 v =
                                *reinterpret_cast<const float4*>(&sinit[(wave * RS + rs) * 32 + c_row(4 * a, lane)]);
                            acc[rs][b][4 * a] = v.x;
                            acc[rs][b][4 * a + 1] = v.y;
                            acc[rs][b][4 * a + 2] = v.z;
                            acc[rs][b][4 * a + 3] = v.w;
                        }
            }
            // the barrier inside also orders the scol writes of chunk s - 1
            // before their sum, and that sum before chunk s + 1 reuses the buffer
            ring_io.advance(ring, s, u, src);
            if (s >= 1) reduce(s - 1);
            chunk_mma_sets<T, D, kKeys, false, RS>(acc, rd, ring + u * G::C::BYTES, qf, kInitLds ? nullptr : c_init,
                                                   kInitLds);
            if (sp.t_begin + (s + 1) * kKeys > P_rows) {  // keys past the range end or inside the causal window
                // key t is visible to window query i (position P_rows + i) iff t - P_rows <= i
#pragma unroll
                for (int rs = 0; rs < RS; ++rs)
#pragma unroll
                    for (int a = 0; a < 4; ++a) {
                        const int4 w4 = *reinterpret_cast<const int4*>(&swin[(wave * RS + rs) * 32 + c_row(4 * a, lane)]);
                        const int wv[4] = {w4.x, w4.y, w4.z, w4.w};
#pragma unroll
                        for (int kb = 0; kb < 2; ++kb) {
                            const int t = sp.t_begin + s * kKeys + 32 * kb + (lane & 31);
#pragma unroll
                            for (int e = 0; e < 4; ++e)
                                if (!(t < sp.t_end && t - P_rows <= wv[e])) acc[rs][kb][4 * a + e] = -INFINITY;
                        }
                    }
            }
            // exponentials of each key block: a lane sum over its 16 rows per set
            // and the other 16 rows from the other half of the wave (a lane
            // swap on the vector unit, not an LDS permute); lane l then writes
            // the sum of key l (block 0 in the lower half, block 1 in the upper)
            float v[2];
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                float c = 0.0f;
#pragma unroll
                for (int rs = 0; rs < RS; ++rs) {
                    f32x16& x = acc[rs][kb];
#pragma unroll
                    for (int i = 0; i < 16; ++i) x[i] = fast_exp2(x[i] * sl2);
                    c += ((x[0] + x[1]) + (x[2] + x[3]) + ((x[4] + x[5]) + (x[6] + x[7]))) +
                         (((x[8] + x[9]) + (x[10] + x[11])) + ((x[12] + x[13]) + (x[14] + x[15])));
                }
                v[kb] = half_wave_sum(c);
            }
            interleave_trans<32 * RS>();
            scol[s & 1][lane][wave] = lane < 32 ? v[0] : v[1];
        }
    }
    __syncthreads();
    reduce(sp.nch - 1);
}

// Pool: one workgroup per (segment, tile of TILE keys).  The tile and its
// halo of h keys on each side are summed over the planes into LDS (TILE / 256
// keys per thread, loads first), then each key takes the max over its window, which
// stops at the end of the candidate prefix; window keys keep their raw score.
// With a role histogram (rh.roles set) the workgroup also counts its candidate
// keys per bucket and top key digit in LDS and adds the non-zero counts to the
// segment's histogram.
// Counting: a tile's candidate keys span few bins (scores of one segment lie
// within a few binades), so the workgroup first finds its lowest bin, counts in
// an LDS window of kRoleHistWindow bins per bucket from there (16-bit halves of
// LDS words) and writes the window as its tile record with plain stores: no
// global atomics, no zero fill, and the latency-bound pool keeps about the LDS,
// and so the residency, it has without counting.  A tile whose bins do not fit
// the window marks its record; the top-k then counts that segment itself.
constexpr int kPoolHistWindow = kRoleHistWindow;

__device__ __forceinline__ uint32_t role_bin(float m) { return score_key(m) >> (32 - kRoleHistBits); }

template <int TILE>
__global__ __launch_bounds__(kThreads) void snap_pool(const float* __restrict__ raw, int planes, int segs,
                                                      int N, int W, int pool_k, int tiles,
                                                      float* __restrict__ score, RoleHist rh, int lab4) {
    __shared__ __align__(16) float ss[TILE + 2 * kMaxPoolHalf + 8];
    extern __shared__ __align__(16) uint32_t lh[];  // [R][kPoolHistWindow / 2] pairs of 16-bit counts when counting
    constexpr int kPoolKeysPerThread = TILE / kThreads;  // consecutive keys per thread
    const int tile = blockIdx.x % tiles;
    const int seg = blockIdx.x / tiles;
    const int h = pool_k / 2;
    const int P = N - W;
    const int t0 = tile * TILE;
    const int n = min(TILE, N - t0) + 2 * h;  // staged keys t0 - h .. t0 + n - h - 1
    const bool counting = rh.roles != nullptr;
    const int8_t* ro = counting ? rh.roles + (size_t)((seg / rh.Hkv) % rh.B) * N : nullptr;
    if (counting)
        for (int e = threadIdx.x; e < rh.R * kPoolHistWindow / 2; e += kThreads) lh[e] = 0u;
    constexpr int kPer = (TILE + 2 * kMaxPoolHalf + kThreads - 1) / kThreads;
    const int e0 = kPoolKeysPerThread * (int)threadIdx.x;
    // labels of this thread's keys, loaded with the sums (their latency hidden
    // behind the pooling): four per word, four-byte loads when rows allow
    uint32_t lab[kPoolKeysPerThread / 4] = {};
    if (counting) {
#pragma unroll
        for (int a = 0; a < kPoolKeysPerThread / 4; ++a) {
            const int t = min(t0 + e0 + 4 * a, N - 4 > 0 ? N - 4 : 0);
            if (lab4) {
                lab[a] = *reinterpret_cast<const uint32_t*>(ro + t);
            } else {
#pragma unroll
                for (int b = 0; b < 4; ++b) lab[a] |= (uint32_t)(uint8_t)ro[min(t0 + e0 + 4 * a + b, N - 1)] << (8 * b);
            }
        }
    }
    float v[kPer];
#pragma unroll
    for (int i = 0; i < kPer; ++i) v[i] = 0.0f;
    for (int pl = 0; pl < planes; ++pl) {
        const float* row = raw + ((size_t)pl * segs + seg) * N;
#pragma unroll
        for (int i = 0; i < kPer; ++i) {  // unconditional loads (clamped index), then the bound
            const int u = t0 - h + i * kThreads + (int)threadIdx.x;
            v[i] += row[min(max(u, 0), N - 1)];
        }
    }
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
        const int e = i * kThreads + (int)threadIdx.x;
        const int u = t0 - h + e;
        if (e < n) ss[e] = (u >= 0 && u < N) ? v[i] : -INFINITY;
    }
    __syncthreads();
    // this thread's kPoolKeysPerThread keys from t0 + e0: pooled values in mv, and the
    // bucket of each candidate (R: not counted) in rv
    float mv[kPoolKeysPerThread];
    uint32_t rv[kPoolKeysPerThread];
    // kernel 7 (the paper's), all windows of this thread inside the prefix:
    // the kPoolKeysPerThread + 6 staged values in registers, the window maxima built from pairwise
    // and four-wide maxima, written as 16-byte stores (rows of a multiple of 4
    // keys keep those aligned)
    const bool fast = h == 3 && (N & 3) == 0 && t0 + e0 + kPoolKeysPerThread - 1 + h < P;
    if (fast) {
        float x[kPoolKeysPerThread + 8];  // staged keys from t0 + e0 - 3 (the last 2 unused)
#pragma unroll
        for (int a = 0; a < (kPoolKeysPerThread + 8) / 4; ++a) {
            const float4 f = *reinterpret_cast<const float4*>(&ss[e0 + 4 * a]);
            x[4 * a] = f.x;
            x[4 * a + 1] = f.y;
            x[4 * a + 2] = f.z;
            x[4 * a + 3] = f.w;
        }
        float p2[kPoolKeysPerThread + 5], p4[kPoolKeysPerThread + 3];
#pragma unroll
        for (int j = 0; j < kPoolKeysPerThread + 5; ++j) p2[j] = fmaxf(x[j], x[j + 1]);
#pragma unroll
        for (int j = 0; j < kPoolKeysPerThread + 3; ++j) p4[j] = fmaxf(p2[j], p2[j + 2]);
        float* dst = score + (size_t)seg * N + t0 + e0;
#pragma unroll
        for (int a = 0; a < kPoolKeysPerThread / 4; ++a) {
#pragma unroll
            for (int b = 0; b < 4; ++b) {
                const int j = 4 * a + b;
                mv[j] = fmaxf(fmaxf(p4[j], p2[j + 4]), x[j + 6]);  // keys j .. j + 6 around key j + 3
            }
            *reinterpret_cast<float4*>(dst + 4 * a) = make_float4(mv[4 * a], mv[4 * a + 1], mv[4 * a + 2],
                                                                  mv[4 * a + 3]);
        }
        if (counting) {
#pragma unroll
            for (int a = 0; a < kPoolKeysPerThread / 4; ++a)
#pragma unroll
                for (int b = 0; b < 4; ++b) rv[4 * a + b] = min((lab[a] >> (8 * b)) & 0xffu, (uint32_t)rh.R);
        }
    } else {
        const int valid = min(TILE, N - t0) - e0;  // keys of this thread inside the row
#pragma unroll
        for (int j = 0; j < kPoolKeysPerThread; ++j) {
            const int t = t0 + e0 + j;
            float m = 0.0f;
            uint32_t r = (uint32_t)rh.R;
            if (j < valid) {
                if (t < P) {
                    const int lo = max(0, t - h), hi = min(P - 1, t + h);
                    m = -INFINITY;
                    for (int u = lo; u <= hi; ++u) m = fmaxf(m, ss[u - t0 + h]);
                    if (counting) r = min((lab[j >> 2] >> (8 * (j & 3))) & 0xffu, (uint32_t)rh.R);
                } else {
                    m = ss[e0 + j + h];
                }
                score[(size_t)seg * N + t] = m;
            }
            mv[j] = m;
            rv[j] = r;
        }
    }
    if (!counting) return;  // uniform
    // the window: the kPoolHistWindow bins up to that of the largest score a
    // segment can have (the G*W window rows' probabilities summed, rh.top); a
    // candidate below it (a score under 2^-117 of that, an exact 0, a NaN)
    // marks the tile, whose segment the top-k then counts itself
    const uint32_t lo = rh.lo;
    bool out_of_window = false;
    uint32_t cur = 0xffffffffu, cnt = 0u;
#pragma unroll
    for (int j = 0; j < kPoolKeysPerThread; ++j) {
        // runs of equal (bucket, bin) along the thread's consecutive keys (the
        // max-pool's plateaus) go in with one atomic: fewer lanes contend for
        // the same LDS word in each atomic instruction
        uint32_t e = 0xffffffffu;
        if (rv[j] < (uint32_t)rh.R) {
            const uint32_t off = role_bin(mv[j]) - lo;
            if (off < (uint32_t)kPoolHistWindow)
                e = rv[j] * kPoolHistWindow + off;
            else
                out_of_window = true;
        }
        if (e != cur) {
            if (cnt != 0u) atomicAdd(&lh[cur >> 1], cnt << (16 * (cur & 1u)));
            cur = e;
            cnt = 0u;
        }
        cnt += e != 0xffffffffu ? 1u : 0u;
    }
    if (cnt != 0u) atomicAdd(&lh[cur >> 1], cnt << (16 * (cur & 1u)));
    const bool fits = !__syncthreads_or(out_of_window);
    // the tile record: header, then the window's count pairs (16-byte stores)
    uint32_t* rec = rh.hist + ((size_t)seg * tiles + tile) * (size_t)(kRoleHistHeader + rh.R * kPoolHistWindow / 2);
    if (threadIdx.x == 0) {
        u32x4 hd = zero16();
        hd.x = lo;
        hd.y = fits ? 0u : 1u;
        st16(rec, hd);
    }
    u32x4* body = reinterpret_cast<u32x4*>(rec + kRoleHistHeader);
    for (int e = threadIdx.x; e < rh.R * kPoolHistWindow / 8; e += kThreads)
        body[e] = fits ? *reinterpret_cast<const u32x4*>(&lh[4 * e]) : zero16();
}

template <typename T, int D, int RS>
void launch_passes(const RowView& qv, const RowView& kv, int B, int Hkv, const float* lse_win, const SnapPlan& p,
                   int N, int W, float sl2, float* stats, float* lse, float* raw, hipStream_t st) {
    const dim3 grid((unsigned)((size_t)p.n_vsegs * p.nranges));
    if (lse_win != nullptr) {  // row statistics from the caller: one read of K
        hipLaunchKernelGGL(snap_import_lse, dim3((unsigned)p.n_vsegs), dim3(p.rpg), 0, st, lse_win, p.rows,
                           p.rgroups, lse);
    } else {
        hipLaunchKernelGGL((snap_pass1<T, D, RS>), grid, dim3(kThreads), 0, st, qv, kv, B, Hkv, N, W, p.rows,
                           p.rgroups, p.nranges, p.range_keys, sl2, stats);
        hipLaunchKernelGGL(snap_combine, dim3((unsigned)p.n_vsegs), dim3(p.rpg * kCombineSplit), 0, st, stats,
                           p.nranges, p.rows,
                           p.rgroups, lse);
    }
    hipLaunchKernelGGL((snap_pass2<T, D, RS>), grid, dim3(kThreads), 0, st, qv, kv, B, Hkv, N, W, p.rows,
                       p.rgroups, p.nranges, p.range_keys, sl2, lse, p.segs, raw);
}

template <typename T, int D>
hipError_t run_snapkv(const RowView& qv, const RowView& kv, const float* lse_win, int L, int B, int Hq, int Hkv,
                      int N, int W, float scale, int pool_k, float* score, const RoleHist& rh, void* ws,
                      hipStream_t st) {
    const SnapPlan p = snap_plan(L, B, Hq, Hkv, N, W, D, (int)sizeof(T));
    char* w = static_cast<char*>(ws);
    float* stats = reinterpret_cast<float*>(w + p.off_stats);
    float* lse = reinterpret_cast<float*>(w + p.off_lse);
    float* raw = reinterpret_cast<float*>(w + p.off_raw);
    const float sl2 = scale * kLog2e;
    if constexpr (sizeof(T) == 2) {
        if (p.sets == 2)
            launch_passes<T, D, 2>(qv, kv, B, Hkv, lse_win, p, N, W, sl2, stats, lse, raw, st);
        else
            launch_passes<T, D, 1>(qv, kv, B, Hkv, lse_win, p, N, W, sl2, stats, lse, raw, st);
    } else {
        launch_passes<T, D, 1>(qv, kv, B, Hkv, lse_win, p, N, W, sl2, stats, lse, raw, st);
    }
    if (rh.roles != nullptr) {
        // label rows 4-byte aligned: the pool reads four labels at a time
        const int lab4 = N % 4 == 0 && (reinterpret_cast<uintptr_t>(rh.roles) & 3u) == 0;
        const int tiles = role_hist_tiles(N);
        const unsigned lds = (unsigned)(rh.R * kPoolHistWindow / 2 * sizeof(uint32_t));
        hipLaunchKernelGGL(snap_pool<kRoleHistTile>, dim3((unsigned)(p.segs * tiles)), dim3(kThreads), lds, st, raw,
                           p.planes, p.segs, N, W, pool_k, tiles, score, rh, lab4);
    } else {
        const int tiles = (N + kPoolTile - 1) / kPoolTile;
        hipLaunchKernelGGL(snap_pool<kPoolTile>, dim3((unsigned)(p.segs * tiles)), dim3(kThreads), 0u, st, raw,
                           p.planes, p.segs, N, W, pool_k, tiles, score, rh, 0);
    }
    return hipGetLastError();
}

}  // namespace

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices];  // device address of `scratch`, per device
}  // namespace

hipError_t snapkv_scratch(void** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch[dev] == nullptr) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (p == nullptr) return hipErrorInvalidSymbol;
        g_scratch[dev] = p;
    }
    *out = g_scratch[dev];
    return hipSuccess;
}

hipError_t launch_snapkv(const RowView& q, const RowView& k, const float* lse_win, int dtype, int L, int B, int Hq,
                         int Hkv, int N, int W, int d, float scale, int pool_k, float* score, const int8_t* roles,
                         int R, uint32_t* hist, void* ws, hipStream_t st) {
    // the largest pooled score is the sum over the G*W window rows of one
    // probability each: the window ends at its bin (+1 for rounding)
    const float top = (float)((Hq / Hkv) * W);
    uint32_t bits;
    std::memcpy(&bits, &top, sizeof(bits));
    const uint32_t top_bin = ((bits | 0x80000000u) >> (32 - kRoleHistBits)) + 1u;
    const RoleHist rh{roles, hist, R, B, Hkv, top_bin >= kRoleHistWindow - 1 ? top_bin + 1u - kRoleHistWindow : 0u};
    if (dtype == 0) {
        if (d == 128)
            return run_snapkv<__bf16, 128>(q, k, lse_win, L, B, Hq, Hkv, N, W, scale, pool_k, score, rh, ws, st);
        return run_snapkv<__bf16, 64>(q, k, lse_win, L, B, Hq, Hkv, N, W, scale, pool_k, score, rh, ws, st);
    }
    if (d == 128)
        return run_snapkv<float, 128>(q, k, lse_win, L, B, Hq, Hkv, N, W, scale, pool_k, score, rh, ws, st);
    return run_snapkv<float, 64>(q, k, lse_win, L, B, Hq, Hkv, N, W, scale, pool_k, score, rh, ws, st);
}

}  // namespace kve
