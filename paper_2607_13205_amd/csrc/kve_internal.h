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
// processed in row groups of 128 (four 32-row blocks, one per wave).  Each
// segment's keys are split into chunks; pass 1 writes per-chunk row softmax
// statistics, a combine step reduces them to one log-sum-exp per row, pass 2
// writes per-row-group column sums, and the pool step adds the row groups and
// max-pools the prefix.
// ---------------------------------------------------------------------------
constexpr int kSnapRowsPerGroup = 128;
constexpr int kSnapTileKeys = 64;
constexpr int kSnapMaxRows = 1024;

struct SnapPlan {
    int segs, rows, rgroups, rows_pad, chunk, nchunks;
    size_t off_stats, off_lse, off_raw, total;
};

inline SnapPlan snap_plan(int L, int B, int Hq, int Hkv, int N, int W) {
    SnapPlan p{};
    p.segs = L * B * Hkv;
    p.rows = (Hq / Hkv) * W;
    p.rgroups = (p.rows + kSnapRowsPerGroup - 1) / kSnapRowsPerGroup;
    p.rows_pad = p.rgroups * kSnapRowsPerGroup;
    // aim for about 2048 workgroups per pass, chunks of 256 .. 4096 keys
    long long want = (long long)N * p.segs * p.rgroups / 2048;
    if (want < 256) want = 256;
    if (want > 4096) want = 4096;
    p.chunk = (int)((want + kSnapTileKeys - 1) / kSnapTileKeys * kSnapTileKeys);
    p.nchunks = (N + p.chunk - 1) / p.chunk;
    size_t off = 0;
    p.off_stats = off;
    off = align_up(off + (size_t)p.segs * p.nchunks * p.rows_pad * 2 * sizeof(float));
    p.off_lse = off;
    off = align_up(off + (size_t)p.segs * p.rows_pad * sizeof(float));
    p.off_raw = off;
    off = align_up(off + (size_t)p.rgroups * p.segs * N * sizeof(float));
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
