// Host-side plans and kernel launchers shared by the C ABI and the HIP sources.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace kve {

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// ---------------------------------------------------------------------------
// SnapKV score: rows of one segment are the G*W window queries (head-major),
// taken in row groups of 128 (a segment and a row group form a vseg).  Each
// vseg's keys are split into ranges; pass 1 writes one log-sum-exp per
// (vseg, range, row), a combine step reduces them to one per row, pass 2 writes
// per-row-group column sums, and the pool step adds the row groups and
// max-pools the prefix.
// ---------------------------------------------------------------------------
constexpr int kSnapRowsPerGroup = 128;
constexpr int kSnapMaxRows = 1024;
constexpr int kSnapMaxRange = 2048;   // keys per workgroup range
constexpr int kFusedChunkKeys = 64;   // keys per item of the persistent path

struct SnapPlan {
    int segs, rows, rgroups, n_vsegs, range_keys, nranges;
    int fchunks_max;  // persistent path: chunks per vseg
    size_t off_err, off_stats, off_lse, off_raw, off_arrive, off_ready, off_fstats, off_flse, total;
};

inline SnapPlan snap_plan(int L, int B, int Hq, int Hkv, int N, int W, int d = 128) {
    (void)d;
    SnapPlan p{};
    p.segs = L * B * Hkv;
    p.rows = (Hq / Hkv) * W;
    p.rgroups = (p.rows + kSnapRowsPerGroup - 1) / kSnapRowsPerGroup;
    p.n_vsegs = p.segs * p.rgroups;
    // about 4096 workgroups per pass, ranges of 256 .. 2048 keys (whole chunks)
    long long want = (long long)N * p.n_vsegs / 4096;
    if (want < 256) want = 256;
    if (want > kSnapMaxRange) want = kSnapMaxRange;
    p.range_keys = (int)((want + kFusedChunkKeys - 1) / kFusedChunkKeys * kFusedChunkKeys);
    p.nranges = (N + p.range_keys - 1) / p.range_keys;
    p.fchunks_max = (N + kFusedChunkKeys - 1) / kFusedChunkKeys;
    size_t off = 0;
    p.off_err = off;  // device status word (first 4 bytes of the workspace)
    off = align_up(off + sizeof(unsigned));
    p.off_stats = off;
    off = align_up(off + (size_t)p.n_vsegs * p.nranges * kSnapRowsPerGroup * sizeof(float));
    p.off_lse = off;
    off = align_up(off + (size_t)p.n_vsegs * kSnapRowsPerGroup * sizeof(float));
    p.off_raw = off;
    off = align_up(off + (size_t)p.rgroups * p.segs * N * sizeof(float));
    p.off_arrive = off;  // persistent path: one completion flag per (vseg, chunk) for each of two phases
    off = align_up(off + (size_t)p.n_vsegs * p.fchunks_max * sizeof(unsigned));
    p.off_ready = off;
    off = align_up(off + (size_t)p.n_vsegs * p.fchunks_max * sizeof(unsigned));
    p.off_fstats = off;
    off = align_up(off + (size_t)p.n_vsegs * p.fchunks_max * kSnapRowsPerGroup * sizeof(float));
    p.off_flse = off;
    off = align_up(off + (size_t)p.n_vsegs * kSnapRowsPerGroup * sizeof(float));
    p.total = off;
    return p;
}

// ---------------------------------------------------------------------------
// H2O score: pass 1 one log-sum-exp per (layer, sample, query head, row);
// pass 2 column sums over the group's heads.
// ---------------------------------------------------------------------------
constexpr int kH2oRowBlock = 128;
constexpr int kH2oKeyBlock = 128;

inline size_t h2o_workspace(int L, int B, int Hq, int N) {
    return align_up((size_t)L * B * Hq * N * sizeof(float));
}

hipError_t launch_snapkv(const void* q, const void* k, int dtype, int L, int B, int Hq, int Hkv,
                         int N, int W, int d, float scale, int pool_k, float* score, void* ws,
                         bool persistent, hipStream_t st);

// Persistent single-read score (raw per-row-group column sums into `raw`).
// Sets *used = false, launching nothing, when the shape does not fit one
// cooperative grid; the caller then runs the two-pass kernels.
hipError_t launch_snapkv_fused(const void* q, const void* k, int dtype, int L, int B, int Hq, int Hkv,
                               int N, int W, int d, float scale, float* raw, void* ws,
                               hipStream_t st, bool* used);

hipError_t launch_h2o(const void* q, const void* k, int dtype, int L, int B, int Hq, int Hkv,
                      int N, int d, float scale, float* score, void* ws, hipStream_t st);

hipError_t launch_topk(const float* score, const int8_t* roles, const int32_t* quota, int L,
                       int B, int Hkv, int N, int W, int R, int k_cap, int32_t* idx_out,
                       int32_t* count_out, hipStream_t st);

hipError_t launch_compact(const void* k, const void* v, int elem_bytes, const int32_t* idx,
                          const int32_t* count, int L, int B, int Hkv, int N, int d, int k_cap,
                          void* k_out, void* v_out, hipStream_t st);

}  // namespace kve
