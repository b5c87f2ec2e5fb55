// Workspace plan of the SnapKV score (shared by its kernels and the C ABI).
#pragma once

#include <stddef.h>

namespace kve {

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// ---------------------------------------------------------------------------
// SnapKV score: rows of one segment are the G*W window queries (head-major),
// taken in row groups (a segment and a row group form a vseg) of 128 rows, or
// of 256 for bf16 when the window has more than 128 rows: a wave then holds
// two sets of 32 rows, so that K is read once per pass for up to 256 rows.  Each
// vseg's keys are split into ranges of whole 64-key chunks, one workgroup each;
// pass 1 writes one log-sum-exp per (vseg, range, row), a combine step reduces
// them to one per row, pass 2 writes the column sums of each row group (a
// plane), and the pool step adds the planes and max-pools the prefix.
// ---------------------------------------------------------------------------
constexpr int kSnapRowsPerGroup = 128;
constexpr int kSnapMaxRows = 1024;
constexpr int kSnapChunkKeys = 64;
constexpr int kSnapTargetGroups = 4096;  // workgroups per pass the range size aims at
constexpr int kSnapMaxRangeChunks = 128;  // at most 8192 keys per range

// Fused role epilogue: per (segment, bucket), the number of candidate
// positions by the top kRoleHistBits bits of their order-preserving score key
// (the top-k's first radix digit), counted by the pool step.  The pool counts
// each tile of kRoleHistTile positions in a window of kRoleHistWindow bins from
// the tile's lowest bin, as 16-bit counts (a tile has fewer than 2^16
// positions); a tile record is a header of four words {lowest bin (all ones:
// no candidate), window overflowed (0/1), 0, 0} and R x kRoleHistWindow / 2
// words of count pairs.  The top-k adds the records of a segment's tiles, or
// counts the segment itself when a tile's bins did not fit its window.
constexpr int kRoleHistBits = 11;
constexpr int kRoleHistBins = 1 << kRoleHistBits;
constexpr int kRoleHistMaxR = 8;
constexpr int kRoleHistTile = 4096;
constexpr int kRoleHistWindow = 512;
constexpr int kRoleHistHeader = 4;

inline size_t role_hist_tile_words(int R) { return (size_t)kRoleHistHeader + (size_t)R * kRoleHistWindow / 2; }
inline int role_hist_tiles(int N) { return (N + kRoleHistTile - 1) / kRoleHistTile; }

// Bytes of the static device scratch array the allocation-free SnapKV entry
// point uses as its workspace (one copy per GPU, held until the process ends).
constexpr size_t kSnapScratchBytes = (size_t)64 << 20;

struct SnapPlan {
    int segs, rows, sets, rpg, rgroups, n_vsegs, range_keys, nranges, planes;
    size_t off_stats, off_lse, off_raw, total;
};

// elem: bytes per element of the inputs (2 for bf16, 4 for fp32)
inline SnapPlan snap_plan(int L, int B, int Hq, int Hkv, int N, int W, int d, int elem) {
    (void)d;
    SnapPlan p{};
    p.segs = L * B * Hkv;
    p.rows = (Hq / Hkv) * W;
    p.sets = (elem == 2 && p.rows > kSnapRowsPerGroup) ? 2 : 1;  // 32-row sets per wave
    p.rpg = p.sets * kSnapRowsPerGroup;                           // rows per row group
    p.rgroups = (p.rows + p.rpg - 1) / p.rpg;
    p.n_vsegs = p.segs * p.rgroups;
    p.planes = p.rgroups;
    // whole chunks per range: about kSnapTargetGroups workgroups per pass, at
    // most 128 chunks each (longer ranges start fewer workgroups, whose query
    // fragments and first chunks are latency before any product), and at least as many
    // keys as the group has query rows (a workgroup loads its rows' queries
    // once, so its keys should outweigh them); short problems thus get short
    // ranges rather than a few workgroups walking many chunks in turn
    const long long chunks = (N + kSnapChunkKeys - 1) / kSnapChunkKeys;
    long long per = (chunks * p.n_vsegs + kSnapTargetGroups - 1) / kSnapTargetGroups;
    const int group_rows = p.rows < p.rpg ? p.rows : p.rpg;
    const long long min_per = (group_rows + kSnapChunkKeys - 1) / kSnapChunkKeys;
    if (per < min_per) per = min_per;
    if (per > kSnapMaxRangeChunks) per = kSnapMaxRangeChunks;
    if (per > chunks) per = chunks;
    p.range_keys = (int)(per * kSnapChunkKeys);
    p.nranges = (int)((chunks + per - 1) / per);
    size_t off = 0;
    p.off_stats = off;
    off = align_up(off + (size_t)p.n_vsegs * p.nranges * p.rpg * sizeof(float));
    p.off_lse = off;
    off = align_up(off + (size_t)p.n_vsegs * p.rpg * sizeof(float));
    p.off_raw = off;
    off = align_up(off + (size_t)p.planes * p.segs * N * sizeof(float));
    p.total = off;
    return p;
}

}  // namespace kve
