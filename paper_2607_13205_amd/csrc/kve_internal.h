// Host-side plans and kernel launchers shared by the C ABI and the HIP sources.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "kve_snap_plan.h"

namespace kve {

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

// ---------------------------------------------------------------------------
// Decode over a compacted cache: the k_cap rows of a segment are cut into
// splits of whole kDecodeQuantum-row quanta, one workgroup each (about
// kDecodeTargetGroups workgroups in all); each writes per head the partial
// output o[d] and its (reference, denominator) pair, merged by a last step.
// ---------------------------------------------------------------------------
constexpr int kDecodeQuantum = 128;
constexpr int kDecodeTargetGroups = 1024;  // one split per segment once there are 1024 segments
constexpr int kDecodeMaxGroup = 8;  // query heads per KV head

struct DecodePlan {
    int segs, G, nsplit, split_keys;
    size_t off_o, off_ml, total;
};

inline DecodePlan decode_plan(int L, int B, int Hq, int Hkv, int k_cap, int d) {
    DecodePlan p{};
    p.segs = L * B * Hkv;
    p.G = Hq / Hkv;
    const long long quanta = (k_cap + kDecodeQuantum - 1) / kDecodeQuantum;
    long long ns = (kDecodeTargetGroups + p.segs - 1) / p.segs;
    if (ns > quanta) ns = quanta;
    if (ns < 1) ns = 1;
    const long long per = (quanta + ns - 1) / ns;
    p.split_keys = (int)(per * kDecodeQuantum);
    p.nsplit = (int)((quanta + per - 1) / per);
    const size_t parts = (size_t)p.segs * p.nsplit * p.G;
    p.off_o = 0;
    p.off_ml = align_up(parts * d * sizeof(float));
    p.total = p.off_ml + align_up(parts * 2 * sizeof(float));
    return p;
}

// ---------------------------------------------------------------------------
// One-shot Quest analogue: a first step writes each head's mean window query
// (the workspace, [segs, G, d] float32); the page step cuts the prefix of a
// segment into pages and gives each workgroup a range of whole wave steps of
// pages (about kQuestTargetGroups workgroups in all).
// ---------------------------------------------------------------------------
constexpr int kQuestTargetGroups = 4096;
constexpr int kQuestMaxGroup = 8;  // query heads per KV head
constexpr int kQuestMaxPage = 1024;

struct QuestPlan {
    int segs, G, n_pages, range_pages, nranges;
    size_t total;
};

inline QuestPlan quest_plan(int L, int B, int Hq, int Hkv, int N, int W, int d, int elem, int page) {
    QuestPlan p{};
    p.segs = L * B * Hkv;
    p.G = Hq / Hkv;
    const int P = N - W;
    p.n_pages = (P + page - 1) / page;
    const int step = 4 * (64 / (d * elem / 16));  // pages per workgroup step: 4 waves
    const long long steps = (p.n_pages + step - 1) / step;
    long long per = (steps * p.segs + kQuestTargetGroups - 1) / kQuestTargetGroups;
    if (per < 1) per = 1;
    p.range_pages = (int)(per * step);
    p.nranges = p.n_pages > 0 ? (int)((p.n_pages + p.range_pages - 1) / p.range_pages) : 1;
    p.total = align_up((size_t)p.segs * p.G * d * sizeof(float));
    return p;
}

// A 4-D view [layer, batch, head, token] of rows of d contiguous elements:
// byte strides of the four dimensions (each a multiple of 16, so that every
// row starts 16-byte aligned).  Dense tensors [L, B, H, T, d] have strides
// (B H T, H T, T, 1) rows of d elements.
struct RowView {
    const char* base;
    long long s_layer, s_batch, s_head, s_token;
};

inline RowView dense_view(const void* p, int B, int H, int T, int d, int elem_bytes) {
    const long long row = (long long)d * elem_bytes;
    return RowView{static_cast<const char*>(p), (long long)B * H * T * row, (long long)H * T * row,
                   (long long)T * row, row};
}

// lse_win: the window rows' natural-log log-sum-exp from the caller, or null
// to compute it (pass 1 and the combine step).  roles: bucket labels [B, N] of
// the fused role epilogue, or null; with them the call also writes the role
// histograms hist [L*B*Hkv, R, kRoleHistBins] (zeroed and filled in the call).
// q: the window queries [L, B, Hq, W, d] as a view (head Hq, token W); k: the
// keys [L, B, Hkv, N, d] as a view.
hipError_t launch_snapkv(const RowView& q, const RowView& k, const float* lse_win, int dtype, int L, int B, int Hq,
                         int Hkv, int N, int W, int d, float scale, int pool_k, float* score, const int8_t* roles,
                         int R, uint32_t* hist, void* ws, hipStream_t st);

// Device address of this GPU's static SnapKV scratch array (kSnapScratchBytes
// bytes), taken once per device with that device current.
hipError_t snapkv_scratch(void** out);

// q: all prefill queries [L, B, Hq, N, d] as a view; k: [L, B, Hkv, N, d] as a view
hipError_t launch_h2o(const RowView& q, const RowView& k, int dtype, int L, int B, int Hq, int Hkv,
                      int N, int d, float scale, float* score, void* ws, hipStream_t st);

// hist: the role histograms of the scores (as the fused SnapKV epilogue writes
// them), or null to count them in a first sweep over the scores
hipError_t launch_topk(const float* score, const int8_t* roles, const int32_t* quota, const uint32_t* hist, int L,
                       int B, int Hkv, int N, int W, int R, int k_cap, int32_t* idx_out,
                       int32_t* count_out, void* ws, hipStream_t st);

hipError_t launch_decode(const void* q, const void* kc, const void* vc, const int32_t* count, int dtype, int L,
                         int B, int Hq, int Hkv, int k_cap, int d, float scale, float* out, void* ws,
                         hipStream_t st);

// q: window queries [L, B, Hq, W, d] as a view; k: keys [L, B, Hkv, N, d] as a view
hipError_t launch_quest(const RowView& q, const RowView& k, int dtype, int L, int B, int Hq, int Hkv, int N, int W,
                        int d, int page, float* score, void* ws, hipStream_t st);

hipError_t launch_probe(const int32_t* ids, int B, int N, const float* weight, const float* bias, int V, int R,
                        int8_t* out, hipStream_t st);

// read-bandwidth probe (measurement helper): `blocks` workgroups stream
// `bytes` (a multiple of 16) once, one value per workgroup written to sink
hipError_t launch_read_probe(const void* buf, size_t bytes, int nontemporal, float* sink, int blocks,
                             hipStream_t st);

// k, v: views [L, B, Hkv, N, d] (v.base null: keys only); outputs dense [L, B, Hkv, k_cap, d]
hipError_t launch_compact(const RowView& k, const RowView& v, int elem_bytes, const int32_t* idx,
                          const int32_t* count, int L, int B, int Hkv, int N, int d, int k_cap,
                          void* k_out, void* v_out, hipStream_t st);

}  // namespace kve
