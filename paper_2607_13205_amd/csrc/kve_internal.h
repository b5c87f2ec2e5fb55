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
// vseg's keys are split into ranges of whole 64-key chunks, one workgroup each;
// pass 1 writes one log-sum-exp per (vseg, range, row), a combine step reduces
// them to one per row, pass 2 writes the column sums of each row group (a
// plane), and the pool step adds the planes and max-pools the prefix.
// ---------------------------------------------------------------------------
constexpr int kSnapRowsPerGroup = 128;
constexpr int kSnapMaxRows = 1024;
constexpr int kSnapChunkKeys = 64;
constexpr int kSnapTargetGroups = 4096;  // workgroups per pass the range size aims at
constexpr int kSnapMaxRangeChunks = 32;  // at most 2048 keys per range

struct SnapPlan {
    int segs, rows, rgroups, n_vsegs, range_keys, nranges, planes;
    size_t off_stats, off_lse, off_raw, total;
};

inline SnapPlan snap_plan(int L, int B, int Hq, int Hkv, int N, int W, int d = 128) {
    (void)d;
    SnapPlan p{};
    p.segs = L * B * Hkv;
    p.rows = (Hq / Hkv) * W;
    p.rgroups = (p.rows + kSnapRowsPerGroup - 1) / kSnapRowsPerGroup;
    p.n_vsegs = p.segs * p.rgroups;
    p.planes = p.rgroups;
    // whole chunks per range: about kSnapTargetGroups workgroups per pass (two
    // per compute unit at a time), 4 .. 32 chunks each (fewer when N is short)
    const long long chunks = (N + kSnapChunkKeys - 1) / kSnapChunkKeys;
    long long per = (chunks * p.n_vsegs + kSnapTargetGroups - 1) / kSnapTargetGroups;
    if (per < 4) per = 4;
    if (per > kSnapMaxRangeChunks) per = kSnapMaxRangeChunks;
    if (per > chunks) per = chunks;
    p.range_keys = (int)(per * kSnapChunkKeys);
    p.nranges = (int)((chunks + per - 1) / per);
    size_t off = 0;
    p.off_stats = off;
    off = align_up(off + (size_t)p.n_vsegs * p.nranges * kSnapRowsPerGroup * sizeof(float));
    p.off_lse = off;
    off = align_up(off + (size_t)p.n_vsegs * kSnapRowsPerGroup * sizeof(float));
    p.off_raw = off;
    off = align_up(off + (size_t)p.planes * p.segs * N * sizeof(float));
    p.total = off;
    return p;
}

// ---------------------------------------------------------------------------
// H2O score: pass 1 one start value (-lse2 / sl2) per (layer, sample, query
// head, row), in rows of pitch h2o_pitch(N) floats; pass 2 one column sum per
// (query head, key), added over the group's heads by a last step.  A pass-1 workgroup covers kH2oRowsPerGroup rows:
// the G heads of a KV group at kH2oRowsPerGroup / G positions.
// ---------------------------------------------------------------------------
constexpr int kH2oRowsPerGroup = 128;

inline int h2o_pitch(int N) { return (N + 63) / 64 * 64; }

// floats before the per-(query head, key) column sums
inline size_t h2o_colsum_offset(int L, int B, int Hq, int N) {
    return align_up((size_t)L * B * Hq * h2o_pitch(N) * sizeof(float)) / sizeof(float);
}

inline size_t h2o_workspace(int L, int B, int Hq, int N) {
    return h2o_colsum_offset(L, B, Hq, N) * sizeof(float) + align_up((size_t)L * B * Hq * N * sizeof(float));
}

hipError_t launch_snapkv(const void* q, const void* k, int dtype, int L, int B, int Hq, int Hkv,
                         int N, int W, int d, float scale, int pool_k, float* score, void* ws,
                         hipStream_t st);

hipError_t launch_h2o(const void* q, const void* k, int dtype, int L, int B, int Hq, int Hkv,
                      int N, int d, float scale, float* score, void* ws, hipStream_t st);

hipError_t launch_topk(const float* score, const int8_t* roles, const int32_t* quota, int L,
                       int B, int Hkv, int N, int W, int R, int k_cap, int32_t* idx_out,
                       int32_t* count_out, hipStream_t st);

hipError_t launch_compact(const void* k, const void* v, int elem_bytes, const int32_t* idx,
                          const int32_t* count, int L, int B, int Hkv, int N, int d, int k_cap,
                          void* k_out, void* v_out, hipStream_t st);

}  // namespace kve
