/*
 * wavefilter.h -- C ABI of the MI355X (gfx950) WaveFilter filter+attend path.
 *
 * WaveFilter (arXiv 2606.00724) replaces attention of a query block over a
 * long cached prompt by attention over a small sparse cache that a
 * coarse-to-fine wavelet search picks, per head:
 *
 *   1. wf_dwt_keys     J-level 1-D DWT of the cached prompt keys along the
 *                      sequence (Section 2.2, eq. 5; Section 3.1, eq. 6).
 *   2. wf_skim_score   perception weights softmax(Q A_J^T * scale) per query
 *                      row (eq. 7), column sums W (eq. 8), top-S coarse
 *                      regions (eq. 9 with the proportion given as a count).
 *   3. wf_scan_select  the regions' tokens (eq. 10) scored the same way at
 *                      token resolution (Section 3.2), top-k tokens -> mu^0.
 *   4. wf_gather_kv    sparse cache [K[mu^0]; K_g], [V[mu^0]; V_g]
 *                      (Section 3.2, last paragraph; Algorithm 1).
 *   5. wf_sparse_attn  attention of the query block over the sparse cache,
 *                      no mask (the cached-attention form of eq. 3).
 *   6. wf_filter_attend  steps 1-5 fused; the sparse cache is never
 *                      materialised.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - A "unit" is one (batch, head) pair; units are independent.  Tensors are
 *    row-major and contiguous, unit-major, with the head dimension d fastest:
 *        Q  [batch][heads][q_len][d]        K, V [batch][heads][ctx_len][d]
 *        Kg, Vg [batch][heads][gen_len][d]  O    [batch][heads][q_len][d]
 *  - Element type of Q, K, V, Kg, Vg, Ks, Vs and O is params->dtype
 *    (WF_BF16 or WF_F32).  Coefficients, scores and all softmax arithmetic
 *    are fp32; index outputs are int32.
 *  - Every tensor pointer is device memory owned by the caller, 16-byte
 *    aligned.  The library never allocates, frees or synchronises: kernels are
 *    queued on `stream` (a hipStream_t; NULL = the default stream) and the
 *    call returns before they finish.
 *  - Calls that need scratch memory take a caller-owned device workspace of
 *    at least wf_workspace_bytes(params, op) bytes (256-byte aligned).  Its
 *    contents need no initialisation and are garbage afterwards; two calls
 *    in flight at once must not share one workspace.
 *  - Every argument is checked on the host before anything is queued.  A
 *    rejected call returns a non-zero wf_status, queues nothing and records a
 *    message that wf_last_error() returns (per thread).  The library never
 *    aborts, throws or prints.  A failure reported by the HIP runtime while
 *    queueing returns WF_ERR_HIP.
 *  - Index sets are returned in ascending order.  Selection orders scores
 *    descending and breaks exact ties by the lower index.
 */
#ifndef WAVEFILTER_H
#define WAVEFILTER_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum wf_status {
    WF_OK = 0,
    WF_ERR_INVALID_ARG = 1, /* null/misaligned pointer, size out of range   */
    WF_ERR_UNSUPPORTED = 2, /* valid request this build does not implement  */
    WF_ERR_WORKSPACE = 3,   /* workspace missing or smaller than required   */
    WF_ERR_HIP = 4          /* the HIP runtime reported an error            */
} wf_status;

/* Wavelet families (Section 2.2; the paper uses Haar throughout).
 * Filters are orthonormal and applied in forward phase,
 * A[n] = sum_m g_m y[2n+m], so Haar coefficient j of level J covers tokens
 * 2^J j .. 2^J j + 2^J - 1, the region of eq. 10.
 *   WF_HAAR: g = (1, 1)/sqrt2
 *   WF_DB2:  Daubechies 4-tap, g = (1+r3, 3+r3, 3-r3, 1-r3)/(4 sqrt2)      */
enum { WF_HAAR = 0, WF_DB2 = 1 };

/* Right-end extension of each level's sequence for WF_DB2 (Haar never reads
 * past the end): half-sample symmetric (y[N] = y[N-1], y[N+1] = y[N-2]) or
 * periodic (y[N+i] = y[i]). */
enum { WF_EXT_SYMMETRIC = 0, WF_EXT_PERIODIC = 1 };

/* Element type of the tensors listed above. */
enum { WF_BF16 = 0, WF_F32 = 1 };

/* Operations whose workspace size wf_workspace_bytes reports. */
enum { WF_OP_SKIM = 0, WF_OP_SCAN = 1, WF_OP_ATTN = 2, WF_OP_FUSED = 3,
       WF_OP_CACHED = 4, WF_OP_SHARED = 5 };

/* Remainder.  When L is not a multiple of 2^J, the first
 * Lf = 2^J floor(L / 2^J) positions are filtered (transformed, scored,
 * selected) and the last R = L - Lf positions are always kept: the sparse
 * cache is [K[tok]; K[Lf .. L); K_g] (values likewise), R = 0 for a multiple
 * of 2^J.  The recursion does the same with 2^B. */

/* Limits of this build. */
enum {
    WF_MAX_LEVELS = 10,  /* J                                   */
    WF_MAX_Q_LEN = 256,  /* B, rows of the query block          */
    /* scratch bytes per device of wf_filter_attend_noalloc (32 MiB) */
    WF_NOALLOC_SCRATCH_BYTES = 33554432
};

typedef struct wf_params {
    int32_t batch;    /* >= 1                                                 */
    int32_t heads;    /* >= 1; K/V heads equal query heads                    */
    int32_t ctx_len;  /* L = |I_p|, prompt positions; see the remainder note */
    int32_t head_dim; /* d: 64 or 128                                         */
    int32_t q_len;    /* B = |I~|, query rows: 1 .. WF_MAX_Q_LEN              */
    int32_t gen_len;  /* G = |I_g| >= 0, tail rows always kept (never scored) */
    int32_t levels;   /* J: 1 .. WF_MAX_LEVELS, 2^J <= L                      */
    int32_t wavelet;  /* WF_HAAR or WF_DB2                                    */
    int32_t boundary; /* WF_EXT_* (read for WF_DB2 only)                      */
    int32_t dtype;    /* WF_BF16 or WF_F32                                    */
    int32_t segments; /* S: coarse regions kept, 1 .. L >> J                  */
    int32_t budget;   /* k >= 1: tokens kept; effective k_eff = min(k, S 2^J) */
    float scale;      /* softmax scale for skim, scan and attention;
                         0 selects 1/sqrt(d) (eqs. 1, 3 and 7)                */
} wf_params;

/* Bytes of workspace `op` needs for these parameters (0 if it needs none or
 * the parameters are invalid). */
size_t wf_workspace_bytes(const wf_params* p, int32_t op);

/* k_eff = min(budget, segments * 2^levels), or -1 if p is invalid. */
int32_t wf_effective_budget(const wf_params* p);

/*
 * Step 1 (eqs. 5-6): J-level DWT of the first Lf keys along the sequence.
 *   K        [batch][heads][L][d]                 dtype
 *   approx   [batch][heads][L >> J][d]            fp32 out: A_J
 *   details  nullable; per unit the rows of D_1, then D_2, ... D_J,
 *            [batch][heads][sum_{j=1..J} Lf >> j][d] fp32 out
 */
wf_status wf_dwt_keys(const wf_params* p, const void* K, float* approx,
                      float* details, void* stream);

/*
 * Step 2 (eqs. 7-9): skim weights and the top-S coarse regions.
 *   Q          [batch][heads][B][d]               dtype
 *   approx     [batch][heads][L >> J][d]          fp32 (from wf_dwt_keys)
 *   seg_score  [batch][heads][L >> J]             fp32 out: W
 *   seg_idx    [batch][heads][S]                  int32 out, ascending
 *   workspace  >= wf_workspace_bytes(p, WF_OP_SKIM)
 */
wf_status wf_skim_score(const wf_params* p, const void* Q, const float* approx,
                        float* seg_score, int32_t* seg_idx, void* workspace,
                        size_t workspace_bytes, void* stream);

/*
 * Step 3 (eq. 10, then eqs. 7-9 at token resolution): the pool is the
 * S 2^J tokens of the regions in seg_idx, in ascending order; each pool
 * token gets W'_t = sum over query rows of its softmax weight (softmax over
 * the pool only); the k_eff best tokens are returned.
 *   Q          [batch][heads][B][d]               dtype
 *   K          [batch][heads][L][d]               dtype
 *   seg_idx    [batch][heads][S]                  int32, strictly ascending,
 *                                                 each in [0, L >> J)
 *   tok_score  nullable [batch][heads][S 2^J]     fp32 out: W' in pool order
 *   tok_idx    [batch][heads][k_eff]              int32 out, ascending
 *   workspace  >= wf_workspace_bytes(p, WF_OP_SCAN)
 * Region ids are not range-checked on the device: out-of-range or unsorted
 * ids are undefined behaviour (the host cannot read device memory).
 */
wf_status wf_scan_select(const wf_params* p, const void* Q, const void* K,
                         const int32_t* seg_idx, float* tok_score,
                         int32_t* tok_idx, void* workspace,
                         size_t workspace_bytes, void* stream);

/*
 * Step 4 (Section 3.2, last paragraph): the sparse cache.
 *   K, V       [batch][heads][L][d]               dtype
 *   tok_idx    [batch][heads][k_eff]              int32, each in [0, L)
 *   Kg, Vg     [batch][heads][G][d]               dtype; NULL iff G == 0
 *   Ks, Vs     [batch][heads][k_eff + R + G][d]   dtype out:
 *              rows r < k_eff: K[tok_idx[r]]; then K[Lf .. L) (the R
 *              remainder rows); then the G tail rows
 */
wf_status wf_gather_kv(const wf_params* p, const void* K, const void* V,
                       const int32_t* tok_idx, const void* Kg, const void* Vg,
                       void* Ks, void* Vs, void* stream);

/*
 * Step 5 (eq. 3 form): O = softmax(scale Q Ks^T) Vs over n_kv cache rows,
 * every query row sees every row (bidirectional, no mask).
 *   Q          [batch][heads][B][d]               dtype
 *   Ks, Vs     [batch][heads][n_kv][d]            dtype, n_kv >= 1
 *   O          [batch][heads][B][d]               dtype out (RNE for bf16)
 *   workspace  >= wf_workspace_bytes(p, WF_OP_ATTN) (sized for n_kv up to
 *              k_eff + R + G; a larger n_kv needs the workspace of a params copy
 *              whose budget/segments/gen_len give that many rows)
 */
wf_status wf_sparse_attn(const wf_params* p, const void* Q, const void* Ks,
                         const void* Vs, int32_t n_kv, void* O,
                         void* workspace, size_t workspace_bytes,
                         void* stream);

/*
 * Steps 1-5 fused for one layer of one denoising step.  The DWT never leaves
 * the chip, and attention reads the selected K/V rows in place.
 *   Q [batch][heads][B][d], K, V [batch][heads][L][d], Kg, Vg
 *   [batch][heads][G][d] (NULL iff G == 0)      dtype
 *   O          [batch][heads][B][d]               dtype out
 *   tok_idx    nullable [batch][heads][k_eff]     int32 out: mu^0, ascending
 *   seg_idx    nullable [batch][heads][S]         int32 out: the coarse
 *              regions J_B of eq. 9, ascending
 *   workspace  >= wf_workspace_bytes(p, WF_OP_FUSED)
 */
wf_status wf_filter_attend(const wf_params* p, const void* Q, const void* K,
                           const void* V, const void* Kg, const void* Vg,
                           void* O, int32_t* tok_idx, int32_t* seg_idx,
                           void* workspace, size_t workspace_bytes,
                           void* stream);

/*
 * wf_filter_attend that also records HIP events around its kernels, for
 * per-kernel timing.  events: array of n_events hipEvent_t handles created by
 * the caller (timing enabled); events[0] is recorded before the first kernel
 * and events[i] after the i-th kernel.  wf_filter_attend_kernels() gives the
 * kernel count for these parameters; n_events must be at least that count
 * plus one.  Same results as wf_filter_attend.
 */
wf_status wf_filter_attend_timed(const wf_params* p, const void* Q,
                                 const void* K, const void* V, const void* Kg,
                                 const void* Vg, void* O, int32_t* tok_idx,
                                 int32_t* seg_idx, void* workspace,
                                 size_t workspace_bytes, void* stream,
                                 void** events, int32_t n_events);

/*
 * wf_filter_attend for callers that cannot allocate device memory: code
 * under HIP graph capture, tight serving loops, hosts that forbid
 * allocation.  Same arguments and results as wf_filter_attend, without the
 * workspace: the library's own scratch array of WF_NOALLOC_SCRATCH_BYTES
 * bytes per device (a device-side static, loaded with the library's code on
 * each device it runs on and held until the process ends) takes its place.
 * The call allocates and frees nothing.
 *   Limit: parameters whose fused workspace (wf_workspace_bytes(p,
 *   WF_OP_FUSED)) exceeds WF_NOALLOC_SCRATCH_BYTES are rejected with
 *   WF_ERR_WORKSPACE before anything is queued.
 *   Every call on one device shares that device's scratch, which keeps the
 *   last call's contents (nothing in it needs to start at zero): two calls
 *   whose kernels overlap on one device -- on different streams, or from
 *   different host threads without ordering -- race and give undefined
 *   results.  Calls queued on one stream are ordered and safe.
 */
wf_status wf_filter_attend_noalloc(const wf_params* p, const void* Q,
                                   const void* K, const void* V,
                                   const void* Kg, const void* Vg, void* O,
                                   int32_t* tok_idx, int32_t* seg_idx,
                                   void* stream);

/* Kernels one wf_filter_attend call queues for these parameters, and the
 * name of the i-th one (static strings), or -1 / NULL if p is invalid. */
int32_t wf_filter_attend_kernels(const wf_params* p);
const char* wf_filter_attend_kernel_name(const wf_params* p, int32_t i);

/* ---------------------------------------------------------------------
 * One step with the coarse prompt keys cached across denoising steps.  The
 * cache update of eq. 4 rewrites only the generation rows, so the prompt's
 * level-J approximation A_J (eq. 6) stays valid from step to step: compute
 * it once with wf_dwt_keys and pass it to every later step.  The step then
 * reads A_J ([batch][heads][ctx_len >> levels][d] fp32, as wf_dwt_keys
 * writes it) instead of all of K; K is still read for the pool and the
 * selected rows.  Results are those of wf_filter_attend with that A_J.
 *   approx     device, from wf_dwt_keys with the same params
 *   workspace  >= wf_workspace_bytes(p, WF_OP_CACHED)
 * Other arguments and errors as in wf_filter_attend.
 * --------------------------------------------------------------------- */
wf_status wf_filter_attend_cached(const wf_params* p, const void* Q,
                                  const float* approx, const void* K,
                                  const void* V, const void* Kg,
                                  const void* Vg, void* O, int32_t* tok_idx,
                                  int32_t* seg_idx, void* workspace,
                                  size_t workspace_bytes, void* stream);

/* Same, recording events[i] before kernel i and events[n] after the last
 * (n = wf_filter_attend_cached_kernels(p); n_events >= n + 1). */
wf_status wf_filter_attend_cached_timed(const wf_params* p, const void* Q,
                                        const float* approx, const void* K,
                                        const void* V, const void* Kg,
                                        const void* Vg, void* O,
                                        int32_t* tok_idx, int32_t* seg_idx,
                                        void* workspace,
                                        size_t workspace_bytes, void* stream,
                                        void** events, int32_t n_events);

/* Kernels one cached call queues and the name of the i-th one, or -1 /
 * NULL if p is invalid. */
int32_t wf_filter_attend_cached_kernels(const wf_params* p);
const char* wf_filter_attend_cached_kernel_name(const wf_params* p, int32_t i);

/* ---------------------------------------------------------------------
 * One step with one selection per sequence, shared by all its heads (the
 * layer-shared form of the selection; the per-head form is
 * wf_filter_attend).  Each head scores its own keys as in eqs. 7-8; the
 * column sums W of the heads of a sequence are added before the top-S of
 * eq. 9, which gives the sequence's regions (eq. 10: one pool for all its
 * heads); the scan's W' of every head over that pool are added before the
 * top-k_eff, which gives the sequence's tokens mu^0; every head then
 * attends with its own query rows over its own K/V rows at those tokens,
 * the L mod 2^J remainder rows and its own tail (eq. 3 form).  The sums run
 * over the heads in order.
 *   Q [batch][heads][B][d], K, V [batch][heads][L][d], Kg, Vg
 *   [batch][heads][G][d] (NULL iff G == 0)      dtype
 *   O          [batch][heads][B][d]               dtype out
 *   tok_idx    nullable [batch][k_eff]            int32 out: mu^0, ascending
 *   seg_idx    nullable [batch][S]                int32 out: the regions,
 *              ascending
 *   workspace  >= wf_workspace_bytes(p, WF_OP_SHARED)
 * Every parameter set wf_filter_attend takes is supported: on its
 * token-level path the scan and the attention take the sequence's
 * selections themselves; otherwise the per-unit skim writes W, one select
 * per sequence takes the regions from the heads' sum, the scan's two
 * passes run per unit over them, and one select per sequence takes the
 * tokens from the heads' sum of W'.
 */
wf_status wf_filter_attend_shared(const wf_params* p, const void* Q,
                                  const void* K, const void* V, const void* Kg,
                                  const void* Vg, void* O, int32_t* tok_idx,
                                  int32_t* seg_idx, void* workspace,
                                  size_t workspace_bytes, void* stream);

/* wf_filter_attend_shared with HIP events around its kernels
 * (n = wf_filter_attend_shared_kernels(p); n_events >= n + 1). */
wf_status wf_filter_attend_shared_timed(const wf_params* p, const void* Q,
                                        const void* K, const void* V,
                                        const void* Kg, const void* Vg, void* O,
                                        int32_t* tok_idx, int32_t* seg_idx,
                                        void* workspace,
                                        size_t workspace_bytes, void* stream,
                                        void** events, int32_t n_events);

/* Kernels one shared call queues and the name of the i-th one, or -1 /
 * NULL if p is invalid or outside the token-level path. */
int32_t wf_filter_attend_shared_kernels(const wf_params* p);
const char* wf_filter_attend_shared_kernel_name(const wf_params* p, int32_t i);

/* ---------------------------------------------------------------------
 * Multi-scale recursive filtering (Section 3.2, eqs. 9-11; Algorithm 1,
 * the loop over scales), for the Haar and Daubechies-2 wavelets.  Scale
 * B = p->levels; selection proportions m_b = proportions[b - 1] for
 * b = 1..B (host array of p->levels floats, each in (0, 1]).  Per unit:
 *
 *   mu^B = all Lf filtered positions (Lf as in the remainder note)
 *   for b = B .. 1:
 *     candidates: the n_b coefficients of the b-level DWT of the gathered
 *       keys K[mu^b], taken as one sequence (eq. 11; eq. 6 at b = B):
 *       n_B = Lf / 2^B, n_b = 2 c_{b+1} below.  Coefficient i covers
 *       positions mu^b[2^b i .. 2^b i + 2^b).  For Haar it is the level-b
 *       coefficient of the prompt block holding those positions; for db2 the
 *       filter reads across the joins of the gathered blocks, with the
 *       boundary rule of p at the gathered sequence's right end.
 *     weights: eqs. 7-8 over the n_b candidates only
 *     keep: the c_b best (eq. 9; ties to the lower index), where
 *       c_b = max(1, ceil(m_b * n_b)) evaluated in double from the float
 *       m_b, at most n_b
 *     mu^{b-1}: the positions the kept candidates cover (eq. 10 through
 *       mu^b), ascending
 *   then attention over [K[mu^0]; K[Lf .. L); Kg], values likewise, as in
 *   wf_filter_attend.
 *
 * mu^0 has 2 c_1 positions, ascending.  p->segments and p->budget are not
 * used.
 * --------------------------------------------------------------------- */

/* c_b for every scale into counts[b - 1] (host array of p->levels).
 * INVALID_ARG for a NULL array or a proportion outside (0, 1]. */
wf_status wf_recursion_counts(const wf_params* p, const float* proportions,
                              int32_t* counts);

/* Workspace bytes wf_filter_attend_recursive needs, or 0 for invalid
 * parameters. */
size_t wf_recursive_workspace_bytes(const wf_params* p,
                                    const float* proportions);

/* The recursion and the attention, asynchronous on `stream`.  Q, K, V, Kg,
 * Vg and O as in wf_filter_attend.
 *   tok_idx    nullable [batch][heads][2 c_1]     int32 out: mu^0, ascending
 *   kept_idx   nullable, int32 out: the kept candidates of the scales
 *              b = B .. 2 as prompt block ids at level b (block j covers
 *              positions 2^b j .. 2^b j + 2^b - 1, so mu^{b-1} is the union
 *              of the kept blocks), ascending per unit.  Scale b's ids are
 *              [batch][heads][c_b] starting at element
 *              batch * heads * (c_B + ... + c_{b+1}); the array holds
 *              batch * heads * (c_B + ... + c_2) elements (none when B = 1).
 *   workspace  caller-owned device memory, 256-byte aligned, of at least
 *              wf_recursive_workspace_bytes(p, proportions) bytes.
 * Errors as in wf_filter_attend. */
wf_status wf_filter_attend_recursive(const wf_params* p,
                                     const float* proportions, const void* Q,
                                     const void* K, const void* V,
                                     const void* Kg, const void* Vg, void* O,
                                     int32_t* tok_idx, int32_t* kept_idx,
                                     void* workspace, size_t workspace_bytes,
                                     void* stream);

/* Same, recording events[i] before kernel i and events[n] after the last
 * (n = wf_filter_attend_recursive_kernels(p); n_events >= n + 1). */
wf_status wf_filter_attend_recursive_timed(
    const wf_params* p, const float* proportions, const void* Q, const void* K,
    const void* V, const void* Kg, const void* Vg, void* O, int32_t* tok_idx,
    int32_t* kept_idx, void* workspace, size_t workspace_bytes, void* stream,
    void** events, int32_t n_events);

/* Kernels one recursive call queues (2 per scale, then the attention and
 * its combine) and the name of the i-th one, or -1 / NULL if p is
 * invalid. */
int32_t wf_filter_attend_recursive_kernels(const wf_params* p);
const char* wf_filter_attend_recursive_kernel_name(const wf_params* p,
                                                   int32_t i);

/* Grouped-query attention (g query heads per KV head) needs no entry point
 * of its own: the selection shared by a KV head's g query heads uses W
 * summed over their query rows, which is the selection of the stacked block
 * of g * q_len rows (W is a column sum of row-wise softmaxes), and attention
 * is row-wise.  With the heads of a group adjacent, Q [batch][g * heads_kv]
 * [q_len][d] is already [batch][heads_kv][g * q_len][d]: pass heads =
 * heads_kv and q_len = g * q_len (at most WF_MAX_Q_LEN). */

/* Loads the library's kernels onto the current device and sets up its
 * per-device state, so that no later call stalls for it (otherwise the
 * first call on a device loads what it launches, a few milliseconds of host
 * time during which the GPU waits).  Optional, for callers that want every
 * call to cost the same (serving loops, timing harnesses); call it once per
 * device with that device current.  Synchronous; the library allocates
 * nothing (the HIP runtime places the code in device memory).  May be
 * called again (it then does nothing new).  Returns WF_ERR_HIP if the HIP
 * runtime cannot load the kernels for this device. */
wf_status wf_init(void);

/* Static description of a status code. */
const char* wf_status_str(wf_status s);

/* Detail of the last non-OK return on the calling thread ("" if none). */
const char* wf_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* WAVEFILTER_H */
