/*
 * kve.h -- C ABI of the role-conditional KV-cache eviction library (libkve.so)
 *
 * The library computes, on one MI355X (gfx950) GPU, the eviction path of
 * "Adaptive Filtering of the KV Cache: Diagnosing and Correcting Structural-Role
 * Bias in LLM Inference": the SnapKV windowed attention score with its 1-D
 * max-pool, the H2O accumulated score used as the baseline scorer, the
 * role-conditional budget allocation, the per-role top-k and the compaction of
 * the kept K/V rows into a dense cache.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Every call returns a kve_status_t.  On any error nothing is launched and no
 *   output is written; kve_last_error() returns a message for the calling
 *   thread.  No exception crosses the ABI.
 * - Arguments are validated before any launch.  Device-side contents (role
 *   labels, quotas, indices) cannot be validated on the host without a
 *   synchronisation; the kernels treat out-of-range device values defensively
 *   (documented per call) and never read or write outside the buffers.
 * - Device buffers belong to the caller.  The library never frees or retains
 *   them and performs no device allocation inside these calls: scratch memory
 *   comes from a caller-provided workspace whose size the matching
 *   *_workspace_size() call returns (0 is a valid size; pass NULL then).
 *   Workspaces must be 256-byte aligned (hipMalloc memory is).
 * - All device work is enqueued on `stream` (a hipStream_t; NULL is the
 *   default stream) without host synchronisation.  Calls on different streams
 *   with different workspaces may run concurrently.
 * - Tensors are dense and row-major in the order of their shape; the last
 *   dimension (head_dim d) is contiguous.  Element type is selected by
 *   kve_dtype_t: bfloat16 or float32.  head_dim d must be 64 or 128.
 * - Shapes use L layers, B batch samples, Hq query heads, Hkv KV heads (Hq a
 *   multiple of Hkv, G = Hq / Hkv query heads share KV head h / G), N cached
 *   tokens, W observation-window tokens (the last W positions), R role
 *   buckets (1..8).
 */
#ifndef KVE_H
#define KVE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define KVE_ABI_VERSION 1

typedef enum kve_status {
    KVE_OK = 0,
    KVE_ERR_INVALID_ARG = 1, /* a pointer, size or parameter is invalid        */
    KVE_ERR_UNSUPPORTED = 2, /* dtype / head_dim / size outside what is built  */
    KVE_ERR_WORKSPACE = 3,   /* workspace or output capacity too small         */
    KVE_ERR_HIP = 4          /* the HIP runtime reported an error at launch    */
} kve_status_t;

typedef enum kve_dtype {
    KVE_DTYPE_BF16 = 0,
    KVE_DTYPE_F32 = 1
} kve_dtype_t;

/*
 * Element strides of a 4-D view [layer, batch, head, token] of rows of d
 * contiguous elements.  A dense [L, B, H, T, d] tensor has strides
 * (B*H*T*d, H*T*d, T*d, d); a token-major cache [L, B, T, H, d] seen as
 * [L, B, H, T, d] has (B*T*H*d, T*H*d, d, H*d); a slice of rows keeps its
 * parent's strides.  The strided entry points take a pointer to this struct
 * per input (NULL: dense).  Every stride must be >= 0 with stride times the
 * element size a multiple of 16 bytes, the base pointer 16-byte aligned, and
 * the token stride at most 2^25 bytes; views may overlap (inputs are only
 * read).  The library cannot check that a view stays inside its allocation:
 * that is the caller's part.
 */
typedef struct kve_strides {
    int64_t layer, batch, head, token;
} kve_strides_t;

/* ABI version (KVE_ABI_VERSION of the built library). */
int kve_version(void);

/* SHA-256 (64 hex digits) of the sources and build flags the library was
 * compiled from, as computed by the package's build script; "unknown" for a
 * build that did not supply it.  Static storage, never freed. */
const char* kve_source_hash(void);

/* Message describing the last error returned on the calling thread ("" if none).
 * The pointer stays valid until the next kve_* call on the same thread. */
const char* kve_last_error(void);

/* ------------------------------------------------------------------------- */
/* SnapKV windowed score (paper §2 and §4 "SnapKV mechanism"; Algorithm 1,    */
/* windowed-mass and pooling steps).                                          */
/* ------------------------------------------------------------------------- */

/* Workspace bytes kve_snapkv_score needs for these shapes. */
size_t kve_snapkv_workspace_size(int L, int B, int Hq, int Hkv, int N, int W, int d);

/*
 * For every (layer l, sample b, KV head j) the last W prefill queries of the G
 * query heads of group j attend causally over all N keys (query at position
 * N-W+i sees keys t <= N-W+i), softmax-normalised per query row.  The raw score
 *     s(t) = sum over the G heads and W window queries of p(query -> t)
 * is max-pooled with an odd kernel `pool_k` (stride 1, same length) over the
 * candidate prefix [0, N-W) only; window positions keep their raw score.
 *
 *   q_win  [L, B, Hq, W, d]  window queries (device, dtype)
 *   k      [L, B, Hkv, N, d] keys           (device, dtype)
 *   scale  softmax scale of the logits <q, k>; 0 selects 1/sqrt(d)
 *   pool_k odd, >= 1 (1 disables pooling)
 *   score  [L, B, Hkv, N] float32 output (device)
 *
 * Requires 1 <= W <= N, G*W <= 1024.  Scores are accumulated in float32 from
 * products of the input type; each row's softmax is taken relative to a
 * running reference that is raised to the largest logit seen whenever a
 * partial sum would leave [0, 2^64], so no exponential overflows and the
 * per-chunk sums merge exactly.
 *
 * The workspace (kve_snapkv_workspace_size bytes, 256-byte aligned, owned by
 * the caller) holds per-row statistics and per-key partial sums; its contents
 * on entry do not matter.  Errors: KVE_ERR_INVALID_ARG (null pointers, bad
 * shapes, even pool_k, negative or non-finite scale), KVE_ERR_UNSUPPORTED
 * (d not 64/128, G*W > 1024, grid too large), KVE_ERR_WORKSPACE (too small),
 * KVE_ERR_HIP (launch failure).  Kernels run asynchronously on `stream`.
 */
kve_status_t kve_snapkv_score(const void* q_win, const void* k, kve_dtype_t dtype,
                              int L, int B, int Hq, int Hkv, int N, int W, int d,
                              float scale, int pool_k, float* score,
                              void* workspace, size_t workspace_bytes, void* stream);

/*
 * kve_snapkv_score on strided views of its inputs (kve_strides_t; NULL means
 * dense): q_win as [L, B, Hq, W, d] (for instance the last W rows of the
 * prefill queries [L, B, Hq, N, d], whose strides it keeps) and k as
 * [L, B, Hkv, N, d] (for instance a token-major cache).  Same arithmetic in
 * the same order: the scores are bit-identical to kve_snapkv_score on dense
 * copies of the views.  Errors: as for kve_snapkv_score, and
 * KVE_ERR_INVALID_ARG for strides the view rules above exclude.
 */
kve_status_t kve_snapkv_score_strided(const void* q_win, const kve_strides_t* q_strides,
                                      const void* k, const kve_strides_t* k_strides,
                                      kve_dtype_t dtype, int L, int B, int Hq, int Hkv, int N,
                                      int W, int d, float scale, int pool_k, float* score,
                                      void* workspace, size_t workspace_bytes, void* stream);

/*
 * kve_snapkv_score with the window rows' statistics supplied by the caller:
 * lse_win[l, b, h, i] is the natural-log log-sum-exp of window row i of
 * query head h over its causal keys,
 *   log sum over t <= N-W+i of exp(scale * <q_win[l, b, h, i], k[l, b, j, t]>),
 * which is what a prefill attention kernel returns per query row (the
 * softmax normaliser of §2).  The score then reads K once: the row
 * statistics pass and its combine step are skipped, and the result is that of
 * kve_snapkv_score up to the rounding of the supplied values.  The values
 * must be finite and use the same scale.
 *
 *   lse_win   [L, B, Hq, W] float32 (device)
 *   others    as for kve_snapkv_score (same workspace size)
 *
 * Errors: as for kve_snapkv_score, and KVE_ERR_INVALID_ARG for a null lse_win.
 */
kve_status_t kve_snapkv_score_lse(const void* q_win, const void* k, const float* lse_win,
                                  kve_dtype_t dtype, int L, int B, int Hq, int Hkv, int N,
                                  int W, int d, float scale, int pool_k, float* score,
                                  void* workspace, size_t workspace_bytes, void* stream);

/*
 * kve_snapkv_score for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same kernels and the same result, bit for bit, with the workspace taken
 * from a static device array of kve_snapkv_scratch_bytes() bytes (64 MiB)
 * instead of a caller's buffer.  The call allocates nothing.  Each GPU the
 * library runs on holds its own copy of the array from the library's first
 * use on it until the process ends; its address is taken on the first call
 * on each device (the current device, to which `stream` must belong).
 *
 * Every call on a GPU shares that GPU's array: calls that overlap in time on
 * one GPU (different streams, or host threads enqueueing concurrently) race on
 * it and must be serialised by the caller.  The array's contents on entry do
 * not matter (nothing in it needs to start at zero).
 *
 * Arguments as for kve_snapkv_score, without the workspace.  Errors: as for
 * kve_snapkv_score; KVE_ERR_WORKSPACE when kve_snapkv_workspace_size() of
 * these shapes exceeds kve_snapkv_scratch_bytes() (about 15 layers of a
 * batch-4, 8-KV-head, N = 32768 stack fit; split larger problems by layer);
 * KVE_ERR_HIP when the array's address cannot be obtained.
 */
kve_status_t kve_snapkv_score_noalloc(const void* q_win, const void* k, kve_dtype_t dtype,
                                      int L, int B, int Hq, int Hkv, int N, int W, int d,
                                      float scale, int pool_k, float* score, void* stream);

/* Size in bytes of the static scratch array of kve_snapkv_score_noalloc. */
size_t kve_snapkv_scratch_bytes(void);

/* ------------------------------------------------------------------------- */
/* H2O accumulated score, the baseline scorer (paper §2, H2O family).         */
/* ------------------------------------------------------------------------- */

/* Workspace bytes kve_h2o_score needs for these shapes. */
size_t kve_h2o_workspace_size(int L, int B, int Hq, int Hkv, int N, int d);

/*
 * s(t) = sum over the G query heads of group j and over every prefill query
 * i >= t of the causal softmax probability p_h(i -> t).  No window, no pool.
 *
 *   q      [L, B, Hq, N, d]  all prefill queries (device, dtype)
 *   k      [L, B, Hkv, N, d] keys (device, dtype)
 *   scale  0 selects 1/sqrt(d)
 *   score  [L, B, Hkv, N] float32 output (device)
 *
 * Two passes on the matrix cores: per-row log-sum-exp over the causal row,
 * then column sums per query head, added over the G heads in head order.
 * Requires Hq/Hkv <= 128.  The workspace (kve_h2o_workspace_size bytes,
 * 256-byte aligned, owned by the caller) holds, per (layer, sample, query
 * head), one start value per query row (rows padded to a multiple of 64
 * floats) and one column sum per key; its contents on entry do not matter.
 * Errors: KVE_ERR_INVALID_ARG (null pointers, bad shapes, negative or
 * non-finite scale), KVE_ERR_UNSUPPORTED (d not 64/128, Hq/Hkv > 128, grid
 * too large), KVE_ERR_WORKSPACE (too small), KVE_ERR_HIP (launch failure).
 */
kve_status_t kve_h2o_score(const void* q, const void* k, kve_dtype_t dtype,
                           int L, int B, int Hq, int Hkv, int N, int d, float scale,
                           float* score, void* workspace, size_t workspace_bytes,
                           void* stream);

/*
 * kve_h2o_score on strided views of its inputs (kve_strides_t; NULL means
 * dense): q as [L, B, Hq, N, d] and k as [L, B, Hkv, N, d], e.g. token-major
 * prefill tensors [L, B, N, H, d].  Same arithmetic in the same order: the
 * scores are bit-identical to kve_h2o_score on dense copies.  Errors: as for
 * kve_h2o_score, and KVE_ERR_INVALID_ARG for strides the view rules exclude.
 */
kve_status_t kve_h2o_score_strided(const void* q, const kve_strides_t* q_strides,
                                   const void* k, const kve_strides_t* k_strides,
                                   kve_dtype_t dtype, int L, int B, int Hq, int Hkv, int N,
                                   int d, float scale, float* score, void* workspace,
                                   size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------- */
/* One-shot Quest analogue (paper §4.1 "Query-aware baseline"): page key bounds  */
/* against the mean window query, a second scorer for the same selection.     */
/* ------------------------------------------------------------------------- */

/* Workspace bytes kve_quest_score needs (0 if invalid). */
size_t kve_quest_workspace_size(int L, int B, int Hq, int Hkv, int d);

/*
 * Per (layer l, sample b, KV head j): the candidate prefix [0, N-W) is cut
 * into pages of `page` consecutive tokens, page i = [i*page, min((i+1)*page,
 * N-W)).  With qbar_h the mean of the W window queries of query head h and
 * kmin, kmax the per-channel minimum and maximum of a page's keys, the page
 * score is
 *   sum over the G heads h of group j, sum over channels c of
 *   max(qbar_h[c] * kmin[c], qbar_h[c] * kmax[c]),
 * an upper bound of sum_h <qbar_h, k_t> for every key t of the page (Quest's
 * criterion, made once after prefill).  score[l, b, j, t] is the score of
 * token t's page for t < N-W and +inf for the window.  Fed to
 * kve_topk_select, one bucket keeps whole pages in bound order (ties: the
 * lower page), the last one cut at the budget; role buckets compose as with
 * the other scores.
 *
 *   q_win     [L, B, Hq, W, d] bf16 or fp32 (device), as for kve_snapkv_score
 *   k         [L, B, Hkv, N, d] same dtype (device)
 *   page      tokens per page, 1 .. 1024 (16 is Quest's usual size)
 *   score     [L, B, Hkv, N] float32 (device)
 *   workspace kve_quest_workspace_size bytes, 256-byte aligned, owned by the
 *             caller: the mean window query of every head, [L, B, Hq, d]
 *             float32; contents on entry do not matter.
 *
 * Requires Hq/Hkv <= 8.  Enqueued on `stream`.  Errors: KVE_ERR_INVALID_ARG
 * (null pointers, bad shapes, W outside [1, N], page outside [1, 1024],
 * misaligned workspace), KVE_ERR_UNSUPPORTED (d not 64/128, Hq/Hkv > 8, grid
 * too large), KVE_ERR_WORKSPACE, KVE_ERR_HIP.
 */
kve_status_t kve_quest_score(const void* q_win, const void* k, kve_dtype_t dtype,
                             int L, int B, int Hq, int Hkv, int N, int W, int d, int page,
                             float* score, void* workspace, size_t workspace_bytes,
                             void* stream);

/*
 * kve_quest_score on strided views of its inputs (kve_strides_t; NULL means
 * dense): q_win as [L, B, Hq, W, d] (e.g. the last W rows of the prefill
 * queries) and k as [L, B, Hkv, N, d] (e.g. a token-major cache).  The same
 * arithmetic in the same order: bit-identical to kve_quest_score on dense
 * copies.  Errors: as for kve_quest_score, and KVE_ERR_INVALID_ARG for strides
 * the view rules exclude.
 */
kve_status_t kve_quest_score_strided(const void* q_win, const kve_strides_t* q_strides,
                                     const void* k, const kve_strides_t* k_strides,
                                     kve_dtype_t dtype, int L, int B, int Hq, int Hkv, int N,
                                     int W, int d, int page, float* score, void* workspace,
                                     size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------- */
/* Role-conditional allocation (paper §4.1 role policy; Algorithm 1,          */
/* per-bucket top-k and redistribution steps).  HOST function.                */
/* ------------------------------------------------------------------------- */

/*
 * Per-sample bucket quotas.  With K = min(N, ceil(budget*N)) the kept tokens
 * and K_p = max(0, K - W) the slots left for the candidate prefix [0, N-W),
 * K_p is split over the buckets with alpha_r > 0 and at least one candidate,
 * in proportion to alpha renormalised over those buckets, each quota the
 * ceiling of its share.  A bucket whose share exceeds its candidate
 * population keeps its whole population and the budget it cannot use is
 * re-split the same way over the buckets still open, until no bucket
 * overflows.  Budget left once every positive-weight bucket is full is not
 * spent.  budget >= 1 is the full-cache baseline: every token is kept.
 * Ceilings are taken as ceil(x - 1e-9) to absorb binary64 rounding.
 *
 *   roles     [B, N] int8 labels in [0, R)  (HOST memory)
 *   alpha     [R] weights >= 0 with a positive sum (HOST)
 *   budget    fraction of tokens kept, > 0
 *   quota_out [B, R] int32 (HOST): prefix tokens kept per bucket
 *   kept_out  [B] int32 (HOST): W + sum of the sample's quotas
 *   k_cap_out max over samples of kept_out (HOST, may be NULL)
 *
 * Rejects labels outside [0, R), negative alpha, a zero alpha sum, W > N.
 */
kve_status_t kve_role_allocate(const int8_t* roles, int B, int N, int R,
                               const double* alpha, double budget, int W,
                               int32_t* quota_out, int32_t* kept_out,
                               int32_t* k_cap_out);

/*
 * Fair-eviction quotas (§4.1 "Fair-eviction baseline": the same retention rate
 * for every bucket).  kve_role_allocate with each sample's own bucket
 * populations as the weights, alpha_r = n_r: with P = N - W candidates and
 * K_p as above, bucket r keeps ceil(n_r * K_p / P) of its n_r candidates (no
 * bucket overflows, so there is no redistribution; the quotas may exceed K_p
 * by fewer than R tokens through the ceilings).  A sample with no candidate
 * prefix (W = N) keeps the window only; budget >= 1 keeps every token.
 * Arguments, ownership and errors as for kve_role_allocate, without alpha.
 */
kve_status_t kve_role_allocate_fair(const int8_t* roles, int B, int N, int R,
                                    double budget, int W, int32_t* quota_out,
                                    int32_t* kept_out, int32_t* k_cap_out);

/*
 * Bucket relabelling: out[i] = map[roles[i]] for i < n.  With it the same
 * allocator and top-k express policies over a coarser partition than the
 * labels, e.g. the No-X counterfactual of §4 ("Counterfactual", Table 2):
 * map role X to bucket 1 and every other role to bucket 0, then allocate with
 * alpha = (1, 0), so that the K_p prefix slots go to the best-scoring tokens
 * of any role but X.
 *
 *   roles [n] int8 labels in [0, R_in) (HOST)
 *   map   [R_in] int8 buckets in [0, 8) (HOST)
 *   out   [n] int8 (HOST, may alias roles)
 *
 * Rejects R_in outside [1, 127], map entries outside [0, 8) and labels outside
 * [0, R_in); out is untouched on error.
 */
kve_status_t kve_role_map(const int8_t* roles, size_t n, const int8_t* map, int R_in,
                          int8_t* out);

/*
 * Linear role probe (§6 "Deployment: a linear role probe"): the role label of
 * every token from a multinomial logistic regression over the token ids at
 * t-2 .. t+2, in place of a structural parser.  For token t of sequence b the
 * score of role r is
 *   bias[r] + sum over o = 0..4 of weight[o, ids[b, t + o - 2], r],
 * summed in float32 in that order (bias first), skipping positions outside
 * [0, N) and ids outside [0, V); the label is the argmax, the lowest role on
 * ties.  Labels are in the probe's own role order; kve_role_map turns them
 * into the allocation's buckets.
 *
 *   ids       [B, N] int32 token ids (device)
 *   weight    [5, V, R] float32 (device): one table per offset t-2 .. t+2
 *   bias      [R] float32 (device)
 *   R         roles, 1 .. 8
 *   roles_out [B, N] int8 (device)
 *
 * Enqueued on `stream`.  Errors: KVE_ERR_INVALID_ARG (null pointers,
 * non-positive sizes, R outside [1, 8]), KVE_ERR_UNSUPPORTED (too many
 * tokens), KVE_ERR_HIP.
 */
kve_status_t kve_role_probe(const int32_t* ids, int B, int N, const float* weight,
                            const float* bias, int V, int R, int8_t* roles_out, void* stream);

/* ------------------------------------------------------------------------- */
/* Per-role top-k selection (Algorithm 1, per-bucket top-k).                  */
/* ------------------------------------------------------------------------- */

/* Workspace bytes kve_topk_select needs for these shapes: 8 bytes per
 * position of every segment, L*B*Hkv*N*8 rounded up to 256 (0 when a size is
 * not positive). */
size_t kve_topk_workspace_size(int L, int B, int Hkv, int N, int R);

/*
 * For every (l, b, j) segment: within each bucket r the candidate tokens
 * t < N-W labelled r are ranked by score descending, ties broken by the lower
 * index, and the first quota[b, r] are kept.  The window [N-W, N) is always
 * kept.  The kept indices are written in ascending order.
 *
 *   score     [L, B, Hkv, N] float32 (device).  -0.0 ranks equal to +0.0 and
 *             NaN ranks below every number.
 *   roles     [B, N] int8 (device); labels outside [0, R) are never kept.
 *   quota     [B, R] int32 (device); negative values count as 0 and values
 *             above the bucket's population as the population.
 *   idx_out   [L, B, Hkv, k_cap] int32 (device): entries [0, count) of each
 *             segment are written, the rest left untouched.
 *   count_out [L, B, Hkv] int32 (device, may be NULL): number of kept tokens
 *             of each segment.  A value above k_cap means the output was
 *             truncated to its first k_cap indices (the caller's k_cap was too
 *             small for the quotas it passed).
 *   workspace kve_topk_workspace_size bytes, 256-byte aligned, owned by the
 *             caller: each segment's surely kept positions and threshold-bin
 *             candidates, staged in order; contents on entry do not matter.
 *
 * Enqueued on `stream`.  Errors: KVE_ERR_INVALID_ARG (null pointers,
 * non-positive sizes, W outside [0, N], R outside [1, 8], k_cap < 0,
 * misaligned workspace), KVE_ERR_UNSUPPORTED (too many segments, N > 2^30),
 * KVE_ERR_WORKSPACE (workspace missing or too small), KVE_ERR_HIP.
 */
kve_status_t kve_topk_select(const float* score, const int8_t* roles, const int32_t* quota,
                             int L, int B, int Hkv, int N, int W, int R, int k_cap,
                             int32_t* idx_out, int32_t* count_out,
                             void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------- */
/* Fused role epilogue (§4.1: top-k within each role bucket; Algorithm 1,     */
/* per-bucket top-k): the score's pool step counts what the per-bucket top-k  */
/* would otherwise count in a first sweep over the scores.                    */
/* ------------------------------------------------------------------------- */

/* Bytes of the role histograms of L*B*Hkv segments of N positions and R
 * buckets (0 if invalid). */
size_t kve_role_hist_size(int L, int B, int Hkv, int N, int R);

/*
 * kve_snapkv_score that also counts, for every segment (l, b, j) and bucket r,
 * the candidate positions t < N-W labelled r by the top 11 bits of their
 * pooled score's order-preserving key (sign, exponent and two mantissa bits,
 * -0 counted as +0, NaN below -inf): the first radix digit of the per-bucket
 * top-k, counted in the pool step's epilogue while the pooled scores are in
 * registers.  The counts are kept per tile of 4096 positions, each tile as a
 * record of four header words {lowest bin counted (0xffffffff: none), 1 if the
 * tile's bins spanned more than its 512-bin window, 0, 0} followed by R x 256
 * words holding the 16-bit counts of bins lowest .. lowest + 511 in pairs (low
 * half first); records are ordered [l, b, j, tile].  kve_topk_select_hist adds
 * a segment's records instead of sweeping its scores and labels (and sweeps
 * when a tile overflowed); the kept sets are those of kve_topk_select, bit for
 * bit.
 *
 *   roles  [B, N] int8 bucket labels (device); labels outside [0, R) are not
 *          counted (and never kept by the top-k)
 *   R      buckets, 1 .. 8
 *   hist   kve_role_hist_size bytes (device, 16-byte aligned): written by the
 *          call (its contents on entry do not matter); the rest as for
 *          kve_snapkv_score (same workspace size).
 *
 * Errors: as for kve_snapkv_score; KVE_ERR_INVALID_ARG for null roles or hist,
 * R outside [1, 8] or a misaligned hist.
 */
kve_status_t kve_snapkv_score_hist(const void* q_win, const void* k, kve_dtype_t dtype,
                                   int L, int B, int Hq, int Hkv, int N, int W, int d,
                                   float scale, int pool_k, const int8_t* roles, int R,
                                   float* score, uint32_t* hist,
                                   void* workspace, size_t workspace_bytes, void* stream);

/*
 * kve_topk_select with the first digit's counts supplied: hist is what
 * kve_snapkv_score_hist wrote for these scores, labels, N and R.  The kept
 * indices and counts are those of kve_topk_select on the same scores, bit for
 * bit; counts that do not belong to the scores give an unspecified kept set
 * (never an access outside the buffers).  Arguments and errors as for
 * kve_topk_select, plus hist (kve_role_hist_size bytes, device, 16-byte
 * aligned; KVE_ERR_INVALID_ARG when null or misaligned).
 */
kve_status_t kve_topk_select_hist(const float* score, const int8_t* roles, const int32_t* quota,
                                  const uint32_t* hist, int L, int B, int Hkv, int N, int W, int R,
                                  int k_cap, int32_t* idx_out, int32_t* count_out,
                                  void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------- */
/* K/V compaction: the dense cache of a compacting implementation (§6).      */
/* ------------------------------------------------------------------------- */

/*
 * k_out[l,b,j,m,:] = k[l,b,j,idx[l,b,j,m],:] and the same for v, bit for bit,
 * for m < min(count[l,b,j], k_cap).  Rows at or beyond that are not written.
 * Index values outside [0, N) are skipped (the row is not written).
 *
 *   k, v          [L, B, Hkv, N, d] (device, dtype)
 *   idx           [L, B, Hkv, k_cap] int32 (device)
 *   count         [L, B, Hkv] int32 (device): valid entries of each idx row
 *   k_out, v_out  [L, B, Hkv, k_cap, d] (device, dtype)
 * v and v_out may both be NULL to compact K only.
 */
kve_status_t kve_kv_compact(const void* k, const void* v, kve_dtype_t dtype,
                            const int32_t* idx, const int32_t* count,
                            int L, int B, int Hkv, int N, int d, int k_cap,
                            void* k_out, void* v_out, void* stream);

/*
 * kve_kv_compact reading k and v through strided views [L, B, Hkv, N, d]
 * (kve_strides_t; NULL means dense), e.g. a token-major cache; the outputs
 * are dense as for kve_kv_compact and bit-identical to it on dense copies.
 * Errors: as for kve_kv_compact, and KVE_ERR_INVALID_ARG for strides the view
 * rules exclude.
 */
kve_status_t kve_kv_compact_strided(const void* k, const kve_strides_t* k_strides,
                                    const void* v, const kve_strides_t* v_strides,
                                    kve_dtype_t dtype, const int32_t* idx, const int32_t* count,
                                    int L, int B, int Hkv, int N, int d, int k_cap,
                                    void* k_out, void* v_out, void* stream);

/* ------------------------------------------------------------------------- */
/* Decode through the keep-set (Algorithm 1, last step; §3 "Setup"; §6        */
/* "Systems cost": a compacting implementation attends over the kept rows).   */
/* ------------------------------------------------------------------------- */

/* Workspace bytes kve_decode_attention needs for these shapes (0 if invalid). */
size_t kve_decode_workspace_size(int L, int B, int Hq, int Hkv, int k_cap, int d);

/*
 * One decode query per head over the first count rows of a compacted cache:
 *   out[l, b, h] = sum_t softmax_t(scale * <q[l, b, h], k_c[l, b, j, t]>) v_c[l, b, j, t]
 * over t < n = min(max(count[l, b, j], 0), k_cap), with j = h / (Hq/Hkv)
 * (contiguous groups).  This equals decoding through the keep-mask over the
 * full cache, with evicted positions masked out; a segment with n = 0 gives
 * zeros.  To attend to the new token as well, append its key and value row
 * at position count and pass count + 1.
 *
 *   q         [L, B, Hq, d] bf16 or fp32 (device)
 *   k_c, v_c  [L, B, Hkv, k_cap, d], same dtype (device), e.g. the output of
 *             kve_kv_compact; rows at and beyond n are never used
 *   count     [L, B, Hkv] int32 (device); kve_topk_select's count_out fits
 *   scale     softmax scale; 0 means 1/sqrt(d)
 *   out       [L, B, Hq, d] float32 (device)
 *   workspace kve_decode_workspace_size bytes, 256-byte aligned, owned by the
 *             caller: per (segment, split, head) a partial output row and a
 *             (reference, denominator) pair; contents on entry do not matter.
 *
 * Requires Hq/Hkv <= 8.  Enqueued on `stream`, no host synchronisation.
 * Errors: KVE_ERR_INVALID_ARG (null pointers, bad shapes, negative or
 * non-finite scale, misaligned workspace), KVE_ERR_UNSUPPORTED (d not 64/128,
 * Hq/Hkv > 8, grid too large), KVE_ERR_WORKSPACE, KVE_ERR_HIP.
 */
kve_status_t kve_decode_attention(const void* q, const void* k_c, const void* v_c,
                                  const int32_t* count, kve_dtype_t dtype, int L, int B,
                                  int Hq, int Hkv, int k_cap, int d, float scale, float* out,
                                  void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------- */
/* Measurement helper (not part of the eviction path).                        */
/* ------------------------------------------------------------------------- */

/*
 * Reads `bytes` bytes of device memory at `buf` once, with 16-byte loads
 * (non-temporal when `nontemporal` is non-zero) from `blocks` workgroups of
 * 256 threads striding over the buffer, and writes one float per workgroup,
 * derived from the bytes read, to sink[0 .. blocks).  Timed around a buffer
 * far larger than the last-level cache it gives the streaming HBM read rate
 * the eviction kernels are compared with; repeated over a buffer that fits in
 * the last-level cache, that cache's re-read rate.
 *
 *   buf      device, 16-byte aligned; bytes a positive multiple of 16
 *   sink     device, at least `blocks` floats
 *   blocks   1 .. 65536
 *
 * Enqueued on `stream`.  Errors: KVE_ERR_INVALID_ARG, KVE_ERR_HIP.
 */
kve_status_t kve_read_probe(const void* buf, size_t bytes, int nontemporal, float* sink, int blocks,
                            void* stream);

#ifdef __cplusplus
}
#endif

#endif /* KVE_H */
