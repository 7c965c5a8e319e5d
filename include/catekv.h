/*
 * catekv.h -- C ABI of the CateKV hybrid-KV decode path on MI355X (gfx950).
 *
 * CateKV (ICML 2025) splits the attention heads of a long-context model into
 * "consistent" heads, which attend to a fixed small set of critical tokens
 * chosen at prefill time, and "adaptive" heads, which keep (most of) their
 * KV cache.  This library implements the data-parallel path of that method:
 *
 *   catekv_score_heads      CV head score per KV head      (Section 3.2, Eq. 1-4)
 *   catekv_classify_heads   consistent/adaptive head types (Eq. 5; static identification)
 *   catekv_select_critical  critical chunks per head       (Algorithm 1, pre-filling stage)
 *   catekv_adaptive_budget  chunk budget for retention eta (Algorithm 1, argtopk(C_chunk, n eta))
 *   catekv_compact_kv       dense compact K/V per head     (Algorithm 1, Cache(K, V, i_k, L_obs))
 *   catekv_decode_plan      split-KV work list for a batch (host side, once per request)
 *   catekv_decode_attn      GQA decode over mixed per-head cache lengths
 *                                                         (Algorithm 1, decoding stage)
 *
 * and, around the decoding stage:
 *
 *   catekv_page_bounds      per-page key minima/maxima of adaptive heads
 *   catekv_retrieve_pages   query-aware page retrieval per step
 *                           (Algorithm 1, Retrieval(q, cache_k, cache_v); Section 4, with Quest)
 *   catekv_append_kv        the generated token of each step into every view
 *
 * Conventions shared by every call
 * --------------------------------
 * - Tensor arguments are caller-owned DEVICE pointers unless the name ends in
 *   _host.  Layouts are row-major with the head dimension d innermost and
 *   contiguous; every K/V row is d elements.
 * - dtype selects the storage type of K, V and Q: CATEKV_F32 (float) or
 *   CATEKV_BF16 (bfloat16 bit patterns).  Arithmetic is fp32 (fp64 for the
 *   final CV statistics); every output is fp32 or an integer.
 * - Supported shapes: d == 128, 1 <= Hkv, Hq % Hkv == 0, Hq / Hkv in
 *   {1, 2, 4, 8}.
 * - Device work is enqueued asynchronously on `stream` (a hipStream_t; NULL
 *   means the default stream).  Only catekv_decode_plan blocks the host.
 * - The library never allocates device memory: calls that need scratch take
 *   a caller-owned workspace sized by the matching *_workspace() function.
 *   Workspaces must be 256-byte aligned.  Two calls that overlap in time must
 *   not share a workspace.
 * - Every call validates all arguments BEFORE enqueuing any work.  A status
 *   other than CATEKV_OK means nothing was enqueued and no output was
 *   touched; catekv_last_error() then returns a message (per host thread).
 *   Launch failures report CATEKV_ERR_HIP.  Faults inside a kernel surface
 *   as HIP errors at the caller's next synchronisation.
 */
#ifndef CATEKV_H
#define CATEKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  CATEKV_OK = 0,
  CATEKV_ERR_INVALID_ARG = -1,  /* null pointer, bad size or inconsistent arguments */
  CATEKV_ERR_UNSUPPORTED = -2,  /* valid request outside the supported shapes/dtypes */
  CATEKV_ERR_WORKSPACE = -3,    /* workspace missing, misaligned or too small */
  CATEKV_ERR_HIP = -4           /* a HIP runtime call failed */
} catekv_status;

typedef enum { CATEKV_F32 = 0, CATEKV_BF16 = 1 } catekv_dtype;

/* K and V base pointers of one (sequence, KV head) cache view.  Row t of the
 * view is at k + t * d elements (same for v). */
typedef struct catekv_kv_ptrs {
  const void* k;
  const void* v;
} catekv_kv_ptrs;

/* Host-side descriptor of a decode work list, filled by catekv_decode_plan and
 * passed back to catekv_decode_attn.  Treat as opaque. */
typedef struct catekv_decode_plan_t {
  uint64_t magic;
  int32_t batch, hq, hkv, split_tokens;
  int32_t n_workers, n_segments, n_slots, n_multi;
  int32_t variant, reserved;
  uint64_t segs_off, workers_off, views_off, slots_off, ws_bytes;
  int64_t max_len_total;
} catekv_decode_plan_t;

/* ------------------------------------------------------------------------ */
/* CV head scoring -- Section 3.2, Eq. 1-4.                                  */
/* ------------------------------------------------------------------------ */

/* Workspace bytes for catekv_score_heads with these sizes. */
size_t catekv_score_heads_workspace(int hq, int hkv, int lq, int64_t n,
                                    int64_t l_init, int64_t l_rec);

/* For every KV head h computes the coefficient-of-variation score of its
 * observation matrix:
 *   A   = mean over the G query heads g of group h of
 *         softmax_j( q_rows[g][i] . k[h][l_init + j] / sqrt(d) ),
 *         j over the key range [l_init, n - l_rec), restricted to keys at
 *         positions <= q_pos0 + i when `causal` is non-zero      (Eq. 1)
 *   Phi = alpha * (linearly interpolated k_pct-quantile of all entries of A)
 *   B   = (A >= Phi),  C_j = sum_i B[i][j]                        (Eq. 2-3)
 *   cv  = population-std(C) / mean(C), and 0 when mean(C) == 0      (Eq. 4)
 *
 * q_rows  [hq][lq][d]  observation rows; row i sits at absolute position
 *                      q_pos0 + i (prefill window: q_pos0 = n - lq;
 *                      decode-time calibration rows: q_pos0 >= n).
 * k       [hkv][n][d]  keys of one sequence.
 * cv_out  [hkv] fp32, device.
 * Errors: INVALID_ARG if l_init < 0, l_rec < 0, l_init + l_rec >= n, lq < 1,
 * k_pct outside [0, 1], alpha <= 0, or (causal and q_pos0 < l_init, which
 * would leave a row with no visible key); WORKSPACE if ws is too small. */
int catekv_score_heads(int dtype, const void* q_rows, int64_t q_pos0, const void* k,
                       int hq, int hkv, int lq, int64_t n, int d,
                       int64_t l_init, int64_t l_rec, double k_pct, double alpha, int causal,
                       float* cv_out, void* ws, size_t ws_bytes, void* stream);

/* Head classification -- Eq. 5 and the reference-based static
 * identification of Section 3.2.  Host only, synchronous.
 * cv_host [S][H]: scores of H heads (all layers of a model, flattened) in S
 * reference samples.  In each sample a head is consistent iff its score is
 * strictly above the linearly interpolated r-quantile of that sample's
 * scores.  The result marks the H - 1 - floor((H - 1) r) heads most often
 * consistent (ties: higher mean score, then lower index), which is the Eq. 5
 * count for distinct scores.  is_consistent_host [H] receives 1/0.
 * Errors: INVALID_ARG for null pointers, S < 1, H < 1 or r outside [0, 1). */
int catekv_classify_heads(const float* cv_host, int S, int H, double r,
                          uint8_t* is_consistent_host);

/* ------------------------------------------------------------------------ */
/* Critical-token selection -- Algorithm 1, pre-filling stage.               */
/* ------------------------------------------------------------------------ */

/* Workspace bytes for catekv_select_critical. */
size_t catekv_select_workspace(int hq, int hkv, int l_obs, int64_t n, int cs, int n_sel);

/* For each KV head h = sel_heads_host[s] (s < n_sel):
 *   A       = mean over the G query heads of group h of
 *             softmax_j( q_obs[g][i] . k[h][j] / sqrt(d) ),  j < n' = n - l_obs
 *   C_j     = sum_i A[i][j]
 *   S_c     = max of C_j over chunk c = [c cs, min((c + 1) cs, n'))
 *   idx_out[s][0 .. b_eff) = the b_eff = min(b, ceil(n'/cs)) chunks with the
 *             largest S_c (ties to the lower chunk index), ascending;
 *             entries b_eff .. b-1 are set to -1.
 * q_obs  [hq][l_obs][d]  the last l_obs prefill query rows.
 * k      [hkv][n][d].
 * sel_heads_host [n_sel] distinct KV head ids (host array).
 * idx_out [n_sel][b] int32, device.
 * Errors: INVALID_ARG if l_obs < 1, l_obs >= n, cs < 1, b < 1, n_sel < 1 or a
 * head id is out of range or repeated; WORKSPACE if ws is too small. */
int catekv_select_critical(int dtype, const void* q_obs, const void* k,
                           int hq, int hkv, int l_obs, int64_t n, int d, int cs,
                           const int32_t* sel_heads_host, int n_sel, int b,
                           int32_t* idx_out, void* ws, size_t ws_bytes, void* stream);

/* catekv_select_critical for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same computation and outputs, with the scratch taken from a
 * 16 MiB device array inside the library (one per GPU, held until the process
 * ends) instead of a caller workspace.  It allocates nothing.  Every call on a
 * GPU shares that GPU's array, so calls that overlap in time on one GPU race
 * (even on different streams); the array keeps the last call's contents and
 * nothing in it needs clearing.  16 MiB covers the selection of up to 8 heads
 * at 1M tokens when cs divides 64 (catekv_select_workspace() gives the need).
 * Errors: those of catekv_select_critical; UNSUPPORTED when the selection
 * needs more scratch than the array holds; HIP if the array's device address
 * cannot be obtained. */
int catekv_select_critical_noalloc(int dtype, const void* q_obs, const void* k,
                                   int hq, int hkv, int l_obs, int64_t n, int d, int cs,
                                   const int32_t* sel_heads_host, int n_sel, int b,
                                   int32_t* idx_out, void* stream);

/* Chunk budget of an adaptive head for retention ratio eta (Algorithm 1,
 * adaptive branch, argtopk(C_chunk, n eta)), counted in chunks of the
 * selection range: *b_out = ceil(eta * ceil((n - l_obs) / cs)), eta read as
 * the decimal ratio it stands for (a product within 1e-9 relative of an
 * integer is that integer); eta = 1 keeps every chunk, i.e. the whole cache,
 * and the last l_obs tokens are kept on top, as for consistent heads.  Host
 * only.
 * Pass the result as b to catekv_select_critical and catekv_compact_kv for
 * the adaptive heads (b >= 1 there; eta small enough to give 0 keeps only
 * the window).
 * Errors: INVALID_ARG for a null b_out, l_obs outside [0, n), cs < 1 or eta
 * outside [0, 1]. */
int catekv_adaptive_budget(int64_t n, int l_obs, int cs, double eta, int64_t* b_out);

/* Cache(K, V, i_k, L_obs) of Algorithm 1: for each selected head s, writes the
 * rows of the chunks idx[s][*] (ascending; entries < 0 ignored; the last chunk
 * may be partial) followed by the last l_obs rows k[h][n - l_obs .. n) into
 * k_c[s] (and likewise V into v_c[s]) as one dense run of rows, and stores
 * the run's length in lens_out[sel_heads_host[s]].
 * k, v      [hkv][n][d]
 * idx       [n_sel][b] int32, device, as written by catekv_select_critical
 * k_c, v_c  [n_sel][b * cs + l_obs][d], device (capacity per head)
 * lens_out  int64 device array indexed by KV head id (e.g. one sequence's
 *           row of a [batch][hkv] length table); other entries untouched.
 * l_obs may be 0 here (chunk rows only): with chunk indices over [0, n) from
 * catekv_retrieve_pages this gathers the retrieved pages of a step.
 * Errors: INVALID_ARG for null pointers or the selection errors above (with
 * l_obs >= 0 allowed).  Index values must come from catekv_select_critical
 * with the same n, l_obs, cs, or from catekv_retrieve_pages with l_obs = 0. */
int catekv_compact_kv(int dtype, const void* k, const void* v, int hkv, int64_t n, int d,
                      int cs, int l_obs, const int32_t* sel_heads_host, int n_sel,
                      const int32_t* idx, int b, void* k_c, void* v_c, int64_t* lens_out,
                      void* stream);

/* ------------------------------------------------------------------------ */
/* Hybrid decode attention -- Algorithm 1, decoding stage.                   */
/* ------------------------------------------------------------------------ */

/* Workspace bytes for a decode plan over max_len_host [batch][hkv].
 * split_tokens is the number of tokens each decode workgroup streams; <= 0
 * spreads all tokens over the workgroups the device holds at once (one per
 * compute unit when all views together hold fewer than 2^18 rows). */
size_t catekv_decode_workspace(const int64_t* max_len_host, int batch, int hq, int hkv,
                               int split_tokens);

/* Builds the split-KV work list for upper-bound cache lengths
 * max_len_host [batch][hkv] (full length for adaptive heads, b cs + l_obs for
 * consistent heads), writes it into ws and fills *plan.  All views are laid
 * end to end and cut into equal shares, one per decode workgroup (by default
 * the number of workgroups the current device runs at once, or one per
 * compute unit below 2^18 rows in all), so long and
 * short views balance across compute units.  Blocks until the upload has
 * completed, so max_len_host may be reused on return.  The plan and ws serve
 * every later catekv_decode_attn call with the same shapes; calls sharing a
 * ws must not overlap in time.
 * Errors: INVALID_ARG for null pointers, batch < 1, negative lengths or a
 * length above 2^31 - 1; WORKSPACE if ws is too small; HIP on upload failure. */
int catekv_decode_plan(const int64_t* max_len_host, int batch, int hq, int hkv,
                       int split_tokens, catekv_decode_plan_t* plan,
                       void* ws, size_t ws_bytes, void* stream);

/* One decode step: for every sequence b and query head g (KV head
 * h = g / (hq / hkv)), with L = min(lens[b][h], planned max_len[b][h]):
 *   s_t = scale * q[b][g] . K_{b,h}[t],  t < L
 *   out[b][g] = sum_t softmax(s)_t V_{b,h}[t],  lse[b][g] = log sum_t exp(s_t)
 * and out = 0, lse = -inf when L == 0.
 * q     [batch][hq][d] (dtype)
 * kv    [batch][hkv] catekv_kv_ptrs, device array (views may point into a
 *       full cache or into compact caches; rows beyond L are never used)
 * lens  [batch][hkv] int64, device (read on the device at run time)
 * out   [batch][hq][d] fp32; lse [batch][hq] fp32 or NULL.
 * scale > 0 and finite (1/sqrt(d) for the paper's attention).
 * ws must be the workspace given to catekv_decode_plan for `plan`.
 * Errors: INVALID_ARG if shapes disagree with the plan, pointers are null or
 * scale is not positive and finite; WORKSPACE if ws is too small. */
int catekv_decode_attn(int dtype, const catekv_decode_plan_t* plan, const void* q,
                       const catekv_kv_ptrs* kv, const int64_t* lens,
                       int batch, int hq, int hkv, int d, float scale,
                       float* out, float* lse, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Query-aware retrieval in adaptive heads -- Algorithm 1, decoding stage,    */
/* Retrieval(q, cache_k, cache_v) "all or query-aware"; the page-based        */
/* retrieval (Quest) that Section 4 integrates into the adaptive heads.       */
/* ------------------------------------------------------------------------ */

/* Page metadata of the selected heads' caches: pages are the chunks of cs
 * rows [p cs, min((p + 1) cs, n)), p < n_pages = ceil(n / cs), and
 *   kmin[s][p][j] = min over the page's rows t of K[heads[s]][t][j]
 *   kmax[s][p][j] = max over the same rows,
 * stored in the dtype of K (exact: minima and maxima of stored values).
 * k           [hkv][n][d] (dtype)
 * heads_host  [n_sel] KV head ids, host array, distinct, 1 <= n_sel <= 128
 * kmin, kmax  [n_sel][n_pages][d] (dtype), caller-allocated
 * Errors: INVALID_ARG for null pointers, n < 1, cs < 1 or a bad head list;
 * UNSUPPORTED for d != 128 or n above 2^31 - 1. */
int catekv_page_bounds(int dtype, const void* k, int hkv, int64_t n, int d, int cs,
                       const int32_t* heads_host, int n_sel, void* kmin, void* kmax, void* stream);

/* Workspace bytes of catekv_retrieve_pages. */
size_t catekv_retrieve_workspace(int n_sel, int64_t n_pages);

/* Pages to attend for one decode step of one sequence.  For each selected
 * head h = heads_host[s] with query heads g in [h G, (h + 1) G), G = hq/hkv:
 *   score[p] = max over g of sum_j max(q[g][j] kmin[s][p][j], q[g][j] kmax[s][p][j])
 * (an upper bound of q_g . k over the page's rows), and idx_out[s] holds the
 * n_keep pages with the largest scores (ties to the lower page), ascending,
 * padded with -1 when n_keep > n_pages.  catekv_compact_kv with l_obs = 0,
 * cs and b = n_keep then gathers those pages' rows for catekv_decode_attn.
 * q        [hq][d] (dtype), the step's queries of this sequence
 * kmin, kmax  from catekv_page_bounds for the same heads_host
 * idx_out  [n_sel][n_keep] int32
 * Errors: INVALID_ARG for null pointers, n_pages < 1, n_keep < 1 or a bad
 * head list; UNSUPPORTED for unsupported shapes; WORKSPACE if ws is too small. */
int catekv_retrieve_pages(int dtype, const void* q, const void* kmin, const void* kmax, int hq, int hkv,
                          int64_t n_pages, int d, const int32_t* heads_host, int n_sel, int n_keep,
                          int32_t* idx_out, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Decode-time KV append -- the generation loop around Algorithm 1's decoding */
/* stage.                                                                     */
/* ------------------------------------------------------------------------ */

/* Appends the newest token's key and value to every (sequence, KV head)
 * view.  For each view bh with L = lens[bh] and 0 <= L < capacity[bh]:
 *   K_bh[L] = k_new[bh],  V_bh[L] = v_new[bh],  lens[bh] = L + 1.
 * The token enters the compact cache of a consistent head and the full cache
 * of an adaptive head alike (the decoding stage attends over every token
 * generated so far, and no stage of Algorithm 1 drops one).  A view with
 * L >= capacity[bh] or L < 0 is left unchanged and sets *overflow = 1 when
 * overflow is not NULL; the library never clears *overflow.
 * A decode plan built once with max_len = capacity serves every step of the
 * growing cache: catekv_decode_attn reads lens on the device and never looks
 * past them.  Run on the stream of the decode steps, so that each step sees
 * the tokens appended before it.
 * kv        [batch][hkv] catekv_kv_ptrs, device; each view's rows must be
 *           writable and number capacity[bh]
 * capacity  [batch][hkv] int64, device: rows allocated per view
 * lens      [batch][hkv] int64, device: read and bumped on the device
 * k_new, v_new  [batch][hkv][d] (dtype)
 * overflow  int32, device, or NULL
 * Errors: INVALID_ARG for null pointers, batch < 1, hkv < 1 or d != 128;
 * UNSUPPORTED for an unknown dtype. */
int catekv_append_kv(int dtype, const catekv_kv_ptrs* kv, const int64_t* capacity, int64_t* lens,
                     const void* k_new, const void* v_new, int batch, int hkv, int d,
                     int32_t* overflow, void* stream);

/* Message describing the last failure on the calling host thread. */
const char* catekv_last_error(void);

/* Library version string. */
const char* catekv_version(void);

#ifdef __cplusplus
}
#endif

#endif /* CATEKV_H */
