// C ABI of libkve: argument validation, the host-side role allocation and the
// dispatch to the HIP launchers.  Declarations and contracts: include/kve.h.
#include "../../include/kve.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "kve_internal.h"

namespace {

// The calling thread's last error message.  A plain character array, so that
// the library registers no thread-exit or process-exit destructor.
thread_local char g_error[512];

kve_status_t fail(kve_status_t st, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_error, sizeof(g_error), fmt, ap);
    va_end(ap);
    return st;
}

kve_status_t ok() {
    g_error[0] = '\0';
    return KVE_OK;
}

kve_status_t from_hip(hipError_t e, const char* what) {
    if (e == hipSuccess) return ok();
    return fail(KVE_ERR_HIP, "%s: HIP error %d (%s)", what, (int)e, hipGetErrorString(e));
}

bool aligned(const void* p) { return (reinterpret_cast<uintptr_t>(p) & (kve::kAlign - 1)) == 0; }

constexpr long long kMaxGrid = 2147483647LL;
constexpr double kCeilGuard = 1e-9;

long long ceil_guarded(double x) { return (long long)std::ceil(x - kCeilGuard); }

kve_status_t check_common(const char* fn, int L, int B, int Hq, int Hkv, int N, int d, int dtype) {
    if (L <= 0 || B <= 0 || Hq <= 0 || Hkv <= 0 || N <= 0 || d <= 0)
        return fail(KVE_ERR_INVALID_ARG, "%s: sizes must be positive (L=%d B=%d Hq=%d Hkv=%d N=%d d=%d)",
                    fn, L, B, Hq, Hkv, N, d);
    if (Hq % Hkv != 0)
        return fail(KVE_ERR_INVALID_ARG, "%s: Hq=%d is not a multiple of Hkv=%d", fn, Hq, Hkv);
    if (dtype != KVE_DTYPE_BF16 && dtype != KVE_DTYPE_F32)
        return fail(KVE_ERR_UNSUPPORTED, "%s: unknown dtype %d", fn, dtype);
    if (d != 64 && d != 128)
        return fail(KVE_ERR_UNSUPPORTED, "%s: head_dim %d not built (64 or 128)", fn, d);
    if ((long long)L * B * Hq > kMaxGrid / 4 || N > (1 << 30))
        return fail(KVE_ERR_UNSUPPORTED, "%s: shape too large", fn);
    return KVE_OK;
}

// Checks shared by the allocators: sizes, budget, window and labels.
kve_status_t check_allocation(const char* fn, const int8_t* roles, int B, int N, int R, double budget, int W) {
    if (B <= 0 || N <= 0) return fail(KVE_ERR_INVALID_ARG, "%s: B and N must be positive", fn);
    if (R < 1 || R > 8) return fail(KVE_ERR_INVALID_ARG, "%s: R=%d outside [1, 8]", fn, R);
    if (W < 0 || W > N) return fail(KVE_ERR_INVALID_ARG, "%s: need 0 <= W <= N (W=%d N=%d)", fn, W, N);
    if (!(std::isfinite(budget) && budget > 0.0))
        return fail(KVE_ERR_INVALID_ARG, "%s: budget must be finite and > 0", fn);
    for (size_t i = 0; i < (size_t)B * N; ++i)
        if (roles[i] < 0 || roles[i] >= R)
            return fail(KVE_ERR_INVALID_ARG, "%s: role label %d at %zu outside [0, %d)", fn, (int)roles[i], i,
                        R);
    return KVE_OK;
}

// n[r]: candidate-prefix tokens (t < N - W) of one sample carrying label r.
void bucket_counts(const int8_t* rb, int N, int W, int R, long long* n) {
    for (int r = 0; r < R; ++r) n[r] = 0;
    for (int t = 0; t < N - W; ++t) ++n[rb[t]];
}

// Quotas of one sample (§4.1 role policy, Algorithm 1): the prefix budget
// K - W split in proportion to alpha over the buckets with alpha > 0 and
// tokens; a bucket whose ceiling share exceeds its population keeps its whole
// population and the rest is re-split over the buckets still open.  Returns
// the kept count W + sum(q).  alpha may sum to 0 (no bucket open: nothing of
// the prefix is kept).
int32_t allocate_sample(const long long* n, const double* alpha, int R, double budget, int N, int W,
                        int32_t* q) {
    for (int r = 0; r < R; ++r) q[r] = 0;
    if (budget >= 1.0) {
        // the full-cache baseline keeps every token
        for (int r = 0; r < R; ++r) q[r] = (int32_t)n[r];
        return N;
    }
    long long K = ceil_guarded(budget * (double)N);
    if (K > N) K = N;
    long long rem = K - W;
    if (rem < 0) rem = 0;
    bool open[8];
    for (int r = 0; r < R; ++r) open[r] = alpha[r] > 0.0 && n[r] > 0;
    while (rem > 0) {
        double total = 0.0;
        int n_open = 0;
        for (int r = 0; r < R; ++r)
            if (open[r]) {
                total += alpha[r];
                ++n_open;
            }
        if (n_open == 0) break;
        long long share[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        bool any_full = false;
        for (int r = 0; r < R; ++r)
            if (open[r]) {
                share[r] = ceil_guarded(alpha[r] / total * (double)rem);
                if (share[r] > n[r]) any_full = true;
            }
        if (!any_full) {
            for (int r = 0; r < R; ++r)
                if (open[r]) q[r] = (int32_t)share[r];
            break;
        }
        // buckets that cannot use their share keep all their tokens; the
        // budget they leave is re-split over the buckets still open
        for (int r = 0; r < R; ++r)
            if (open[r] && share[r] > n[r]) {
                q[r] = (int32_t)n[r];
                rem -= n[r];
                open[r] = false;
            }
        if (rem < 0) rem = 0;
    }
    long long sum = W;
    for (int r = 0; r < R; ++r) sum += q[r];
    return (int32_t)sum;
}

// Largest token stride of a view, in bytes: the chunk loads keep the offsets
// of 64 rows in 32 bits.
constexpr long long kMaxTokenStrideBytes = 1LL << 25;

// The view of a [L, B, H, T, d] input: dense when st is null, else checked
// against the view rules of kve.h.
kve_status_t make_view(const char* fn, const char* name, const void* p, const kve_strides_t* st, int B, int H,
                       int T, int d, int es, kve::RowView* out) {
    if (st == nullptr) {
        *out = kve::dense_view(p, B, H, T, d, es);
        return KVE_OK;
    }
    const long long s[4] = {st->layer, st->batch, st->head, st->token};
    for (int i = 0; i < 4; ++i) {
        if (s[i] < 0) return fail(KVE_ERR_INVALID_ARG, "%s: %s has a negative stride", fn, name);
        if (s[i] > (1LL << 40)) return fail(KVE_ERR_INVALID_ARG, "%s: %s stride too large", fn, name);
        if ((s[i] * es) % 16 != 0)
            return fail(KVE_ERR_INVALID_ARG, "%s: %s stride %lld is not a multiple of 16 bytes", fn, name, s[i]);
    }
    if (s[3] * es > kMaxTokenStrideBytes)
        return fail(KVE_ERR_INVALID_ARG, "%s: %s token stride of %lld bytes exceeds %lld", fn, name, s[3] * es,
                    kMaxTokenStrideBytes);
    if ((reinterpret_cast<uintptr_t>(p) & 15u) != 0)
        return fail(KVE_ERR_INVALID_ARG, "%s: %s not 16-byte aligned", fn, name);
    *out = kve::RowView{static_cast<const char*>(p), s[0] * es, s[1] * es, s[2] * es, s[3] * es};
    return KVE_OK;
}

// use_scratch: the workspace is this GPU's static scratch array (workspace
// and workspace_bytes are ignored); the plan must fit in it
// roles/R/hist: the fused role epilogue (roles == nullptr: none)
// q_st/k_st: strides of the inputs' views (null: dense)
kve_status_t snapkv_common(const char* fn, const void* q_win, const void* k, const float* lse_win,
                           kve_dtype_t dtype, int L, int B, int Hq, int Hkv, int N, int W, int d, float scale,
                           int pool_k, float* score, void* workspace, size_t workspace_bytes, void* stream,
                           bool use_scratch = false, const int8_t* roles = nullptr, int R = 0,
                           uint32_t* hist = nullptr, const kve_strides_t* q_st = nullptr,
                           const kve_strides_t* k_st = nullptr) {
    kve_status_t st = check_common(fn, L, B, Hq, Hkv, N, d, (int)dtype);
    if (st != KVE_OK) return st;
    if (q_win == nullptr || k == nullptr || score == nullptr)
        return fail(KVE_ERR_INVALID_ARG, "%s: null tensor pointer", fn);
    const int es = dtype == KVE_DTYPE_BF16 ? 2 : 4;
    kve::RowView qv, kv;
    if ((st = make_view(fn, "q_win", q_win, q_st, B, Hq, W, d, es, &qv)) != KVE_OK) return st;
    if ((st = make_view(fn, "k", k, k_st, B, Hkv, N, d, es, &kv)) != KVE_OK) return st;
    if (W < 1 || W > N) return fail(KVE_ERR_INVALID_ARG, "%s: need 1 <= W <= N (W=%d N=%d)", fn, W, N);
    if (pool_k < 1 || pool_k % 2 == 0 || pool_k > 255)
        return fail(KVE_ERR_INVALID_ARG, "%s: pool_k must be odd in [1, 255] (got %d)", fn, pool_k);
    if (!(std::isfinite(scale) && scale >= 0.0f))
        return fail(KVE_ERR_INVALID_ARG, "%s: scale must be finite and >= 0", fn);
    if (roles != nullptr) {
        if (hist == nullptr) return fail(KVE_ERR_INVALID_ARG, "%s: null hist", fn);
        if (R < 1 || R > kve::kRoleHistMaxR)
            return fail(KVE_ERR_INVALID_ARG, "%s: R=%d outside [1, %d]", fn, R, kve::kRoleHistMaxR);
        if ((reinterpret_cast<uintptr_t>(hist) & 15u) != 0)
            return fail(KVE_ERR_INVALID_ARG, "%s: hist not 16-byte aligned", fn);
    }
    const long long rows = (long long)(Hq / Hkv) * W;
    if (rows > kve::kSnapMaxRows)
        return fail(KVE_ERR_UNSUPPORTED, "%s: G*W=%lld exceeds %d", fn, rows, kve::kSnapMaxRows);
    const kve::SnapPlan p = kve::snap_plan(L, B, Hq, Hkv, N, W, d, dtype == KVE_DTYPE_BF16 ? 2 : 4);
    if ((long long)p.n_vsegs * p.nranges > kMaxGrid)
        return fail(KVE_ERR_UNSUPPORTED, "%s: shape too large", fn);
    if (use_scratch) {
        if (p.total > kve::kSnapScratchBytes)
            return fail(KVE_ERR_WORKSPACE,
                        "%s: these shapes need %zu bytes of workspace, above the %zu-byte static scratch "
                        "(call kve_snapkv_score with a workspace, or fewer layers per call)",
                        fn, p.total, kve::kSnapScratchBytes);
        const hipError_t e = kve::snapkv_scratch(&workspace);
        if (e != hipSuccess) return from_hip(e, fn);
    } else {
        if (workspace_bytes < p.total || (p.total > 0 && workspace == nullptr))
            return fail(KVE_ERR_WORKSPACE, "%s: workspace of %zu bytes < %zu needed", fn, workspace_bytes,
                        p.total);
        if (!aligned(workspace)) return fail(KVE_ERR_INVALID_ARG, "%s: workspace not 256-byte aligned", fn);
    }
    if (scale == 0.0f) scale = 1.0f / std::sqrt((float)d);
    return from_hip(kve::launch_snapkv(qv, kv, lse_win, (int)dtype, L, B, Hq, Hkv, N, W, d, scale, pool_k,
                                       score, roles, R, hist, workspace, static_cast<hipStream_t>(stream)),
                    fn);
}

// Checks of kve_topk_select and its fused-histogram variant.
kve_status_t topk_common(const char* fn, const float* score, const int8_t* roles, const int32_t* quota,
                         const uint32_t* hist, bool want_hist, int L, int B, int Hkv, int N, int W, int R,
                         int k_cap, int32_t* idx_out, int32_t* count_out, void* workspace, size_t workspace_bytes,
                         void* stream) {
    if (score == nullptr || roles == nullptr || quota == nullptr)
        return fail(KVE_ERR_INVALID_ARG, "%s: null pointer", fn);
    if (want_hist && hist == nullptr) return fail(KVE_ERR_INVALID_ARG, "%s: null hist", fn);
    if (want_hist && (reinterpret_cast<uintptr_t>(hist) & 15u) != 0)
        return fail(KVE_ERR_INVALID_ARG, "%s: hist not 16-byte aligned", fn);
    if (L <= 0 || B <= 0 || Hkv <= 0 || N <= 0)
        return fail(KVE_ERR_INVALID_ARG, "%s: sizes must be positive", fn);
    if (W < 0 || W > N) return fail(KVE_ERR_INVALID_ARG, "%s: need 0 <= W <= N", fn);
    if (R < 1 || R > 8) return fail(KVE_ERR_INVALID_ARG, "%s: R=%d outside [1, 8]", fn, R);
    if (k_cap < 0) return fail(KVE_ERR_INVALID_ARG, "%s: k_cap < 0", fn);
    if (k_cap > 0 && idx_out == nullptr) return fail(KVE_ERR_INVALID_ARG, "%s: null idx_out", fn);
    if ((long long)L * B * Hkv > kMaxGrid || N > (1 << 30))
        return fail(KVE_ERR_UNSUPPORTED, "%s: shape too large", fn);
    const size_t need = kve::align_up((size_t)L * B * Hkv * N * 8);
    if (workspace_bytes < need || workspace == nullptr)
        return fail(KVE_ERR_WORKSPACE, "%s: workspace of %zu bytes < %zu needed", fn, workspace_bytes, need);
    if (!aligned(workspace)) return fail(KVE_ERR_INVALID_ARG, "%s: workspace not 256-byte aligned", fn);
    return from_hip(kve::launch_topk(score, roles, quota, want_hist ? hist : nullptr, L, B, Hkv, N, W, R, k_cap,
                                     idx_out, count_out, workspace, static_cast<hipStream_t>(stream)),
                    fn);
}

// Checks of kve_kv_compact and its strided variant.
kve_status_t compact_common(const char* fn, const void* k, const kve_strides_t* k_st, const void* v,
                            const kve_strides_t* v_st, kve_dtype_t dtype, const int32_t* idx,
                            const int32_t* count, int L, int B, int Hkv, int N, int d, int k_cap, void* k_out,
                            void* v_out, void* stream) {
    if (k == nullptr || idx == nullptr || count == nullptr || k_out == nullptr)
        return fail(KVE_ERR_INVALID_ARG, "%s: null pointer", fn);
    if ((v == nullptr) != (v_out == nullptr))
        return fail(KVE_ERR_INVALID_ARG, "%s: v and v_out must both be given or both be NULL", fn);
    if (L <= 0 || B <= 0 || Hkv <= 0 || N <= 0 || k_cap < 0)
        return fail(KVE_ERR_INVALID_ARG, "%s: invalid sizes", fn);
    if (dtype != KVE_DTYPE_BF16 && dtype != KVE_DTYPE_F32)
        return fail(KVE_ERR_UNSUPPORTED, "%s: unknown dtype %d", fn, (int)dtype);
    if (d != 64 && d != 128) return fail(KVE_ERR_UNSUPPORTED, "%s: head_dim %d not built", fn, d);
    const long long segs = (long long)L * B * Hkv;
    if (segs * ((k_cap + 63) / 64) > kMaxGrid) return fail(KVE_ERR_UNSUPPORTED, "%s: shape too large", fn);
    const int es = dtype == KVE_DTYPE_BF16 ? 2 : 4;
    kve::RowView kv, vv{};
    kve_status_t st = make_view(fn, "k", k, k_st, B, Hkv, N, d, es, &kv);
    if (st != KVE_OK) return st;
    if (v != nullptr && (st = make_view(fn, "v", v, v_st, B, Hkv, N, d, es, &vv)) != KVE_OK) return st;
    return from_hip(kve::launch_compact(kv, vv, es, idx, count, L, B, Hkv, N, d, k_cap, k_out, v_out,
                                        static_cast<hipStream_t>(stream)),
                    fn);
}

// Checks of kve_h2o_score and its strided variant.
kve_status_t h2o_common(const char* fn, const void* q, const kve_strides_t* q_st, const void* k,
                        const kve_strides_t* k_st, kve_dtype_t dtype, int L, int B, int Hq, int Hkv, int N, int d,
                        float scale, float* score, void* workspace, size_t workspace_bytes, void* stream) {
    kve_status_t st = check_common(fn, L, B, Hq, Hkv, N, d, (int)dtype);
    if (st != KVE_OK) return st;
    if (q == nullptr || k == nullptr || score == nullptr)
        return fail(KVE_ERR_INVALID_ARG, "%s: null tensor pointer", fn);
    const int es = dtype == KVE_DTYPE_BF16 ? 2 : 4;
    kve::RowView qv, kv;
    if ((st = make_view(fn, "q", q, q_st, B, Hq, N, d, es, &qv)) != KVE_OK) return st;
    if ((st = make_view(fn, "k", k, k_st, B, Hkv, N, d, es, &kv)) != KVE_OK) return st;
    if (!(std::isfinite(scale) && scale >= 0.0f))
        return fail(KVE_ERR_INVALID_ARG, "%s: scale must be finite and >= 0", fn);
    const int G = Hq / Hkv;
    if (G > kve::kH2oRowsPerGroup)
        return fail(KVE_ERR_UNSUPPORTED, "%s: Hq/Hkv=%d exceeds %d", fn, G, kve::kH2oRowsPerGroup);
    const long long nblk = (N + kve::kH2oRowsPerGroup / G - 1) / (kve::kH2oRowsPerGroup / G);
    const long long nkb = (N + 127) / 128;  // pass-2 key blocks
    if ((long long)L * B * Hkv * nblk > kMaxGrid || (long long)L * B * Hq * nkb > kMaxGrid)
        return fail(KVE_ERR_UNSUPPORTED, "%s: shape too large", fn);
    const size_t need = kve::h2o_workspace(L, B, Hq, N);
    if (workspace_bytes < need || workspace == nullptr)
        return fail(KVE_ERR_WORKSPACE, "%s: workspace of %zu bytes < %zu needed", fn, workspace_bytes, need);
    if (!aligned(workspace)) return fail(KVE_ERR_INVALID_ARG, "%s: workspace not 256-byte aligned", fn);
    if (scale == 0.0f) scale = 1.0f / std::sqrt((float)d);
    return from_hip(kve::launch_h2o(qv, kv, (int)dtype, L, B, Hq, Hkv, N, d, scale, score, workspace,
                                    static_cast<hipStream_t>(stream)),
                    fn);
}

// Checks of kve_quest_score and its strided variant.
kve_status_t quest_common(const char* fn, const void* q_win, const kve_strides_t* q_st, const void* k,
                          const kve_strides_t* k_st, kve_dtype_t dtype, int L, int B, int Hq, int Hkv, int N, int W,
                          int d, int page, float* score, void* workspace, size_t workspace_bytes, void* stream) {
    kve_status_t st = check_common(fn, L, B, Hq, Hkv, N, d, (int)dtype);
    if (st != KVE_OK) return st;
    if (q_win == nullptr || k == nullptr || score == nullptr)
        return fail(KVE_ERR_INVALID_ARG, "%s: null tensor pointer", fn);
    const int es = dtype == KVE_DTYPE_BF16 ? 2 : 4;
    kve::RowView qv, kv;
    if ((st = make_view(fn, "q_win", q_win, q_st, B, Hq, W, d, es, &qv)) != KVE_OK) return st;
    if ((st = make_view(fn, "k", k, k_st, B, Hkv, N, d, es, &kv)) != KVE_OK) return st;
    if (W < 1 || W > N) return fail(KVE_ERR_INVALID_ARG, "%s: need 1 <= W <= N (W=%d N=%d)", fn, W, N);
    if (page < 1 || page > kve::kQuestMaxPage)
        return fail(KVE_ERR_INVALID_ARG, "%s: page must be in [1, %d] (got %d)", fn, kve::kQuestMaxPage, page);
    if (Hq / Hkv > kve::kQuestMaxGroup)
        return fail(KVE_ERR_UNSUPPORTED, "%s: Hq/Hkv=%d exceeds %d", fn, Hq / Hkv, kve::kQuestMaxGroup);
    const kve::QuestPlan p = kve::quest_plan(L, B, Hq, Hkv, N, W, d, dtype == KVE_DTYPE_BF16 ? 2 : 4, page);
    if ((long long)p.segs * p.nranges > kMaxGrid) return fail(KVE_ERR_UNSUPPORTED, "%s: shape too large", fn);
    if (workspace_bytes < p.total || workspace == nullptr)
        return fail(KVE_ERR_WORKSPACE, "%s: workspace of %zu bytes < %zu needed", fn, workspace_bytes,
                    p.total);
    if (!aligned(workspace)) return fail(KVE_ERR_INVALID_ARG, "%s: workspace not 256-byte aligned", fn);
    return from_hip(kve::launch_quest(qv, kv, (int)dtype, L, B, Hq, Hkv, N, W, d, page, score, workspace,
                                      static_cast<hipStream_t>(stream)),
                    fn);
}

}  // namespace

extern "C" {

int kve_version(void) { return KVE_ABI_VERSION; }

#ifndef KVE_SOURCE_HASH
#define KVE_SOURCE_HASH "unknown"
#endif
const char* kve_source_hash(void) { return KVE_SOURCE_HASH; }

const char* kve_last_error(void) { return g_error; }

size_t kve_snapkv_workspace_size(int L, int B, int Hq, int Hkv, int N, int W, int d) {
    if (L <= 0 || B <= 0 || Hq <= 0 || Hkv <= 0 || N <= 0 || W <= 0 || Hq % Hkv != 0) return 0;
    if (d != 64 && d != 128) return 0;
    // the layout differs by dtype: enough for either
    const size_t a = kve::snap_plan(L, B, Hq, Hkv, N, W, d, 2).total;
    const size_t b = kve::snap_plan(L, B, Hq, Hkv, N, W, d, 4).total;
    return a > b ? a : b;
}

kve_status_t kve_snapkv_score(const void* q_win, const void* k, kve_dtype_t dtype, int L, int B,
                              int Hq, int Hkv, int N, int W, int d, float scale, int pool_k,
                              float* score, void* workspace, size_t workspace_bytes, void* stream) {
    return snapkv_common("kve_snapkv_score", q_win, k, nullptr, dtype, L, B, Hq, Hkv, N, W, d, scale, pool_k,
                         score, workspace, workspace_bytes, stream);
}

kve_status_t kve_snapkv_score_strided(const void* q_win, const kve_strides_t* q_strides, const void* k,
                                      const kve_strides_t* k_strides, kve_dtype_t dtype, int L, int B, int Hq,
                                      int Hkv, int N, int W, int d, float scale, int pool_k, float* score,
                                      void* workspace, size_t workspace_bytes, void* stream) {
    return snapkv_common("kve_snapkv_score_strided", q_win, k, nullptr, dtype, L, B, Hq, Hkv, N, W, d, scale,
                         pool_k, score, workspace, workspace_bytes, stream, false, nullptr, 0, nullptr, q_strides,
                         k_strides);
}

kve_status_t kve_snapkv_score_lse(const void* q_win, const void* k, const float* lse_win, kve_dtype_t dtype,
                                  int L, int B, int Hq, int Hkv, int N, int W, int d, float scale, int pool_k,
                                  float* score, void* workspace, size_t workspace_bytes, void* stream) {
    if (lse_win == nullptr) return fail(KVE_ERR_INVALID_ARG, "kve_snapkv_score_lse: null lse_win");
    return snapkv_common("kve_snapkv_score_lse", q_win, k, lse_win, dtype, L, B, Hq, Hkv, N, W, d, scale,
                         pool_k, score, workspace, workspace_bytes, stream);
}

kve_status_t kve_snapkv_score_noalloc(const void* q_win, const void* k, kve_dtype_t dtype, int L, int B, int Hq,
                                      int Hkv, int N, int W, int d, float scale, int pool_k, float* score,
                                      void* stream) {
    return snapkv_common("kve_snapkv_score_noalloc", q_win, k, nullptr, dtype, L, B, Hq, Hkv, N, W, d, scale,
                         pool_k, score, nullptr, 0, stream, true);
}

size_t kve_snapkv_scratch_bytes(void) { return kve::kSnapScratchBytes; }

size_t kve_h2o_workspace_size(int L, int B, int Hq, int Hkv, int N, int d) {
    (void)Hkv;
    (void)d;
    if (L <= 0 || B <= 0 || Hq <= 0 || N <= 0) return 0;
    return kve::h2o_workspace(L, B, Hq, N);
}


kve_status_t kve_h2o_score(const void* q, const void* k, kve_dtype_t dtype, int L, int B, int Hq,
                           int Hkv, int N, int d, float scale, float* score, void* workspace,
                           size_t workspace_bytes, void* stream) {
    return h2o_common("kve_h2o_score", q, nullptr, k, nullptr, dtype, L, B, Hq, Hkv, N, d, scale, score, workspace,
                      workspace_bytes, stream);
}

kve_status_t kve_h2o_score_strided(const void* q, const kve_strides_t* q_strides, const void* k,
                                   const kve_strides_t* k_strides, kve_dtype_t dtype, int L, int B, int Hq,
                                   int Hkv, int N, int d, float scale, float* score, void* workspace,
                                   size_t workspace_bytes, void* stream) {
    return h2o_common("kve_h2o_score_strided", q, q_strides, k, k_strides, dtype, L, B, Hq, Hkv, N, d, scale,
                      score, workspace, workspace_bytes, stream);
}

kve_status_t kve_role_allocate(const int8_t* roles, int B, int N, int R, const double* alpha,
                               double budget, int W, int32_t* quota_out, int32_t* kept_out,
                               int32_t* k_cap_out) {
    const char* fn = "kve_role_allocate";
    if (roles == nullptr || alpha == nullptr || quota_out == nullptr || kept_out == nullptr)
        return fail(KVE_ERR_INVALID_ARG, "%s: null pointer", fn);
    kve_status_t st = check_allocation(fn, roles, B, N, R, budget, W);
    if (st != KVE_OK) return st;
    double asum = 0.0;
    for (int r = 0; r < R; ++r) {
        if (!(std::isfinite(alpha[r]) && alpha[r] >= 0.0))
            return fail(KVE_ERR_INVALID_ARG, "%s: alpha[%d] must be finite and >= 0", fn, r);
        asum += alpha[r];
    }
    if (!(asum > 0.0)) return fail(KVE_ERR_INVALID_ARG, "%s: alpha sums to 0", fn);
    std::vector<int32_t> quota((size_t)B * R, 0), kept(B, 0);
    int32_t k_cap = 0;
    for (int b = 0; b < B; ++b) {
        long long n[8];
        bucket_counts(roles + (size_t)b * N, N, W, R, n);
        kept[b] = allocate_sample(n, alpha, R, budget, N, W, quota.data() + (size_t)b * R);
        if (kept[b] > k_cap) k_cap = kept[b];
    }
    for (size_t i = 0; i < quota.size(); ++i) quota_out[i] = quota[i];
    for (int b = 0; b < B; ++b) kept_out[b] = kept[b];
    if (k_cap_out != nullptr) *k_cap_out = k_cap;
    return ok();
}

kve_status_t kve_role_allocate_fair(const int8_t* roles, int B, int N, int R, double budget, int W,
                                    int32_t* quota_out, int32_t* kept_out, int32_t* k_cap_out) {
    const char* fn = "kve_role_allocate_fair";
    if (roles == nullptr || quota_out == nullptr || kept_out == nullptr)
        return fail(KVE_ERR_INVALID_ARG, "%s: null pointer", fn);
    kve_status_t st = check_allocation(fn, roles, B, N, R, budget, W);
    if (st != KVE_OK) return st;
    std::vector<int32_t> quota((size_t)B * R, 0), kept(B, 0);
    int32_t k_cap = 0;
    for (int b = 0; b < B; ++b) {
        long long n[8];
        bucket_counts(roles + (size_t)b * N, N, W, R, n);
        // each bucket weighted by its own population: the same share of every bucket
        double alpha[8];
        for (int r = 0; r < R; ++r) alpha[r] = (double)n[r];
        kept[b] = allocate_sample(n, alpha, R, budget, N, W, quota.data() + (size_t)b * R);
        if (kept[b] > k_cap) k_cap = kept[b];
    }
    for (size_t i = 0; i < quota.size(); ++i) quota_out[i] = quota[i];
    for (int b = 0; b < B; ++b) kept_out[b] = kept[b];
    if (k_cap_out != nullptr) *k_cap_out = k_cap;
    return ok();
}

kve_status_t kve_role_map(const int8_t* roles, size_t n, const int8_t* map, int R_in, int8_t* out) {
    const char* fn = "kve_role_map";
    if ((n > 0 && (roles == nullptr || out == nullptr)) || map == nullptr)
        return fail(KVE_ERR_INVALID_ARG, "%s: null pointer", fn);
    if (R_in < 1 || R_in > 127) return fail(KVE_ERR_INVALID_ARG, "%s: R_in=%d outside [1, 127]", fn, R_in);
    for (int r = 0; r < R_in; ++r)
        if (map[r] < 0 || map[r] >= 8)
            return fail(KVE_ERR_INVALID_ARG, "%s: map[%d]=%d outside [0, 8)", fn, r, (int)map[r]);
    for (size_t i = 0; i < n; ++i)
        if (roles[i] < 0 || roles[i] >= R_in)
            return fail(KVE_ERR_INVALID_ARG, "%s: role label %d at %zu outside [0, %d)", fn, (int)roles[i], i,
                        R_in);
    for (size_t i = 0; i < n; ++i) out[i] = map[roles[i]];
    return ok();
}

size_t kve_quest_workspace_size(int L, int B, int Hq, int Hkv, int d) {
    if (L <= 0 || B <= 0 || Hq <= 0 || Hkv <= 0 || Hq % Hkv != 0) return 0;
    if (d != 64 && d != 128) return 0;
    return kve::align_up((size_t)L * B * Hq * d * sizeof(float));
}

kve_status_t kve_quest_score(const void* q_win, const void* k, kve_dtype_t dtype, int L, int B, int Hq,
                             int Hkv, int N, int W, int d, int page, float* score, void* workspace,
                             size_t workspace_bytes, void* stream) {
    return quest_common("kve_quest_score", q_win, nullptr, k, nullptr, dtype, L, B, Hq, Hkv, N, W, d, page, score,
                        workspace, workspace_bytes, stream);
}

kve_status_t kve_quest_score_strided(const void* q_win, const kve_strides_t* q_strides, const void* k,
                                     const kve_strides_t* k_strides, kve_dtype_t dtype, int L, int B, int Hq,
                                     int Hkv, int N, int W, int d, int page, float* score, void* workspace,
                                     size_t workspace_bytes, void* stream) {
    return quest_common("kve_quest_score_strided", q_win, q_strides, k, k_strides, dtype, L, B, Hq, Hkv, N, W, d,
                        page, score, workspace, workspace_bytes, stream);
}

size_t kve_decode_workspace_size(int L, int B, int Hq, int Hkv, int k_cap, int d) {
    if (L <= 0 || B <= 0 || Hq <= 0 || Hkv <= 0 || k_cap <= 0 || Hq % Hkv != 0) return 0;
    if (d != 64 && d != 128) return 0;
    return kve::decode_plan(L, B, Hq, Hkv, k_cap, d).total;
}

kve_status_t kve_decode_attention(const void* q, const void* k_c, const void* v_c, const int32_t* count,
                                  kve_dtype_t dtype, int L, int B, int Hq, int Hkv, int k_cap, int d,
                                  float scale, float* out, void* workspace, size_t workspace_bytes,
                                  void* stream) {
    const char* fn = "kve_decode_attention";
    kve_status_t st = check_common(fn, L, B, Hq, Hkv, k_cap, d, (int)dtype);
    if (st != KVE_OK) return st;
    if (q == nullptr || k_c == nullptr || v_c == nullptr || count == nullptr || out == nullptr)
        return fail(KVE_ERR_INVALID_ARG, "%s: null tensor pointer", fn);
    if (!(std::isfinite(scale) && scale >= 0.0f))
        return fail(KVE_ERR_INVALID_ARG, "%s: scale must be finite and >= 0", fn);
    if (Hq / Hkv > kve::kDecodeMaxGroup)
        return fail(KVE_ERR_UNSUPPORTED, "%s: Hq/Hkv=%d exceeds %d", fn, Hq / Hkv, kve::kDecodeMaxGroup);
    const kve::DecodePlan p = kve::decode_plan(L, B, Hq, Hkv, k_cap, d);
    if ((long long)p.segs * p.nsplit > kMaxGrid)
        return fail(KVE_ERR_UNSUPPORTED, "%s: shape too large", fn);
    if (workspace_bytes < p.total || workspace == nullptr)
        return fail(KVE_ERR_WORKSPACE, "%s: workspace of %zu bytes < %zu needed", fn, workspace_bytes,
                    p.total);
    if (!aligned(workspace)) return fail(KVE_ERR_INVALID_ARG, "%s: workspace not 256-byte aligned", fn);
    if (scale == 0.0f) scale = 1.0f / std::sqrt((float)d);
    return from_hip(kve::launch_decode(q, k_c, v_c, count, (int)dtype, L, B, Hq, Hkv, k_cap, d, scale, out,
                                       workspace, static_cast<hipStream_t>(stream)),
                    fn);
}

kve_status_t kve_role_probe(const int32_t* ids, int B, int N, const float* weight, const float* bias, int V,
                            int R, int8_t* roles_out, void* stream) {
    const char* fn = "kve_role_probe";
    if (ids == nullptr || weight == nullptr || bias == nullptr || roles_out == nullptr)
        return fail(KVE_ERR_INVALID_ARG, "%s: null pointer", fn);
    if (B <= 0 || N <= 0 || V <= 0) return fail(KVE_ERR_INVALID_ARG, "%s: B, N and V must be positive", fn);
    if (R < 1 || R > 8) return fail(KVE_ERR_INVALID_ARG, "%s: R=%d outside [1, 8]", fn, R);
    if ((long long)B * N > (long long)kMaxGrid * 256) return fail(KVE_ERR_UNSUPPORTED, "%s: shape too large", fn);
    return from_hip(kve::launch_probe(ids, B, N, weight, bias, V, R, roles_out, static_cast<hipStream_t>(stream)),
                    fn);
}

size_t kve_topk_workspace_size(int L, int B, int Hkv, int N, int R) {
    (void)R;
    if (L <= 0 || B <= 0 || Hkv <= 0 || N <= 0) return 0;
    // one staged (position, tag) pair of 8 bytes per position of every segment
    return kve::align_up((size_t)L * B * Hkv * N * 8);
}

kve_status_t kve_topk_select(const float* score, const int8_t* roles, const int32_t* quota, int L,
                             int B, int Hkv, int N, int W, int R, int k_cap, int32_t* idx_out,
                             int32_t* count_out, void* workspace, size_t workspace_bytes,
                             void* stream) {
    return topk_common("kve_topk_select", score, roles, quota, nullptr, false, L, B, Hkv, N, W, R, k_cap, idx_out,
                       count_out, workspace, workspace_bytes, stream);
}

kve_status_t kve_topk_select_hist(const float* score, const int8_t* roles, const int32_t* quota,
                                  const uint32_t* hist, int L, int B, int Hkv, int N, int W, int R, int k_cap,
                                  int32_t* idx_out, int32_t* count_out, void* workspace, size_t workspace_bytes,
                                  void* stream) {
    return topk_common("kve_topk_select_hist", score, roles, quota, hist, true, L, B, Hkv, N, W, R, k_cap, idx_out,
                       count_out, workspace, workspace_bytes, stream);
}

size_t kve_role_hist_size(int L, int B, int Hkv, int N, int R) {
    if (L <= 0 || B <= 0 || Hkv <= 0 || N <= 0 || R < 1 || R > kve::kRoleHistMaxR) return 0;
    return (size_t)L * B * Hkv * kve::role_hist_tiles(N) * kve::role_hist_tile_words(R) * sizeof(uint32_t);
}

kve_status_t kve_snapkv_score_hist(const void* q_win, const void* k, kve_dtype_t dtype, int L, int B, int Hq,
                                   int Hkv, int N, int W, int d, float scale, int pool_k, const int8_t* roles, int R,
                                   float* score, uint32_t* hist, void* workspace, size_t workspace_bytes,
                                   void* stream) {
    if (roles == nullptr) return fail(KVE_ERR_INVALID_ARG, "kve_snapkv_score_hist: null roles");
    return snapkv_common("kve_snapkv_score_hist", q_win, k, nullptr, dtype, L, B, Hq, Hkv, N, W, d, scale, pool_k,
                         score, workspace, workspace_bytes, stream, false, roles, R, hist);
}


kve_status_t kve_kv_compact(const void* k, const void* v, kve_dtype_t dtype, const int32_t* idx,
                            const int32_t* count, int L, int B, int Hkv, int N, int d, int k_cap,
                            void* k_out, void* v_out, void* stream) {
    return compact_common("kve_kv_compact", k, nullptr, v, nullptr, dtype, idx, count, L, B, Hkv, N, d, k_cap,
                          k_out, v_out, stream);
}

kve_status_t kve_kv_compact_strided(const void* k, const kve_strides_t* k_strides, const void* v,
                                    const kve_strides_t* v_strides, kve_dtype_t dtype, const int32_t* idx,
                                    const int32_t* count, int L, int B, int Hkv, int N, int d, int k_cap,
                                    void* k_out, void* v_out, void* stream) {
    return compact_common("kve_kv_compact_strided", k, k_strides, v, v_strides, dtype, idx, count, L, B, Hkv, N,
                          d, k_cap, k_out, v_out, stream);
}

kve_status_t kve_read_probe(const void* buf, size_t bytes, int nontemporal, float* sink, int blocks,
                            void* stream) {
    const char* fn = "kve_read_probe";
    if (buf == nullptr || sink == nullptr) return fail(KVE_ERR_INVALID_ARG, "%s: null pointer", fn);
    if (bytes == 0 || bytes % 16 != 0)
        return fail(KVE_ERR_INVALID_ARG, "%s: bytes must be a positive multiple of 16", fn);
    if ((reinterpret_cast<uintptr_t>(buf) & 15u) != 0)
        return fail(KVE_ERR_INVALID_ARG, "%s: buffer not 16-byte aligned", fn);
    if (blocks < 1 || blocks > 65536) return fail(KVE_ERR_INVALID_ARG, "%s: blocks outside [1, 65536]", fn);
    return from_hip(kve::launch_read_probe(buf, bytes, nontemporal, sink, blocks, static_cast<hipStream_t>(stream)),
                    fn);
}

}  // extern "C"
