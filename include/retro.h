/*
 * retro.h — C ABI of an MI355X (gfx950) library for one decode step of
 * retrospective sparse attention ("Retrospective Sparse Attention for
 * Efficient Long-Context Generation", Alg. 1 without its UpdateKV step).
 *
 * One step of one attention layer, for a batch of sequences:
 *   1. append the step's key/value to a paged KV cache and keep per-page key
 *      min/max digests (Sec. 2.1, "Dynamic Sparse Attention");
 *   2. score every page against the current query, eq. (quest_score), and keep
 *      the top-k pages under a token budget (PageSelect);
 *   3. record, per KV head and page, the last step the page was loaded, and hand
 *      the previous value to the attention kernel (Alg. 2, UpdateAndBuildMask);
 *   4. one attention pass over the selected pages for the current query and the
 *      W past queries of the retrospective window, a past query taking only the
 *      pages it has not seen (eq. update-org, eq. update-sup, "Retrospective
 *      Mask" paragraph);
 *   5. merge the past queries' supplementary outputs into an output cache of
 *      (output, log-sum-exp) per past query, eq. (merged_attn_general), and
 *      return the finished output of the query leaving the window.
 *
 * Window convention: W counts PAST queries.  A step processes W+1 queries:
 * row r of the window is the query of step tau = t - W + r, row W the current
 * one.  (The paper's window w counts the current query too: W = w - 1.)
 * W = 0 is plain query-aware sparse attention without retrospection.
 *
 * Conventions for every entry point
 *   - All buffers are caller-owned DEVICE memory, contiguous, row-major, with
 *     the layouts given below.  The library allocates nothing and keeps no state
 *     between calls; scratch lives in the caller's `workspace`.
 *   - Work is enqueued on `stream` (a hipStream_t; NULL = the default stream)
 *     and is asynchronous: no call synchronises the host.
 *   - Argument errors are detected on the host before anything is enqueued and
 *     return RETRO_EINVAL / RETRO_EUNSUPPORTED / RETRO_EWORKSPACE; a failed
 *     launch returns RETRO_EHIP.  No C++ exception crosses the ABI.
 *   - Device-side contract (not checkable on the host): seq_lens, page_table,
 *     selections and the mask hold values produced by this library or obeying
 *     the ranges documented here.  Out-of-range page numbers are skipped by the
 *     kernels instead of being dereferenced.
 *   - Calls that share buffers must be ordered by the caller (same stream).
 */
#ifndef RETRO_H
#define RETRO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  RETRO_OK = 0,
  RETRO_EINVAL = -1,        /* null pointer, negative size, inconsistent dimension */
  RETRO_EUNSUPPORTED = -2,  /* well-formed but outside the supported shapes */
  RETRO_EHIP = -3,          /* a HIP launch or query failed */
  RETRO_EWORKSPACE = -4,    /* workspace null or smaller than retro_workspace_size() */
  RETRO_ESCRATCH = -5       /* retro_step_noalloc: the step needs more than the library's
                               static scratch, or a clear of it would be captured */
} retro_status;

typedef enum { RETRO_F32 = 0, RETRO_BF16 = 1 } retro_dtype;

/* Bits of retro_dims.flags.  0 lets retro_step choose its launches (the normal
 * case); the other bits select a launch sequence explicitly or test the failure
 * path, with the same results. */
typedef enum {
  /* retro_step: the page scores take a launch of their own even where the
   * scores, selection and attention fit in one launch */
  RETRO_FLAG_SEPARATE_SCORES = 1,
  /* retro_step: the selection runs at the end of the score launch (implies a
   * separate score launch) */
  RETRO_FLAG_SELECT_IN_SCORES = 2,
  /* tests of the failure path only: every bounded wait between the workgroups
   * of a launch gives up after a few polls, as if its producers never came */
  RETRO_FLAG_TEST_WAIT_TIMEOUT = 4
} retro_flag;

/* Problem statement of one layer.  Supported: head_dim 64 or 128; page_size
 * 16 or 32; 1 <= group <= 16; 0 <= window <= 64; (window+1)*group <= 1024;
 * page_size <= budget_tokens; 0 <= budget_permille <= 1000; max_pages <= 16384;
 * flags a combination of retro_flag bits. */
typedef struct retro_dims {
  int32_t batch;           /* sequences in the batch                                   */
  int32_t num_kv_heads;    /* h_k                                                      */
  int32_t group;           /* G query heads per KV head; h_q = h_k * G (GQA)            */
  int32_t head_dim;        /* d                                                        */
  int32_t page_size;       /* P tokens per page                                        */
  int32_t budget_tokens;   /* B; each step keeps k = min(B_t / P, pages of the sequence) */
  int32_t window;          /* W past queries revisited per step                        */
  int32_t max_pages;       /* length of a page-table row (logical pages per sequence)  */
  int32_t num_phys_pages;  /* physical pages in k_cache / v_cache / digest             */
  int32_t dtype;           /* retro_dtype of queries, keys, values and digests         */
  float sm_scale;          /* softmax scale applied to q.k; 0 selects 1/sqrt(d)         */
  int32_t budget_permille; /* relative budget (Sec. 4 ablation; Table 1's setting of
                              0.15 = 150): B_t = max(B, floor(L * budget_permille /
                              1000)) tokens for a sequence of L tokens (the step's
                              token included); 0: B_t = B.  k_max covers the largest
                              B_t of a full page-table row.                          */
  int32_t flags;           /* retro_flag bits; 0 for normal use                        */
  int32_t reuse_interval;  /* top-k selection reuse, the baseline of the paper's
                              motivational study (Appendix, Table 4) as an alternative
                              PageSelect: with f = reuse_interval >= 2, steps t with
                              t mod f != 0 keep the selection (rows and counts) that
                              `sel` holds from the previous step, unscored, and run
                              UpdateAndBuildMask (Alg. 2) on it; steps with t mod f
                              == 0 select as usual.  0 or 1: every step selects.    */
} retro_dims;

/* The paged KV cache of one layer (Sec. 2.1; pages as in a vLLM-style pool).
 *   k_cache     [num_phys_pages][h_k][P][d]   dtype  key page, token-major
 *   v_cache     [num_phys_pages][h_k][d][P]   dtype  value page, stored transposed
 *                                                    (d-major) so that the token
 *                                                    contraction reads contiguously
 *   digest      [batch][h_k][max_pages][2][d] dtype  per LOGICAL page of each sequence:
 *                                                    [0] = element-wise key minimum,
 *                                                    [1] = maximum over the page's
 *                                                    stored tokens (Quest digest); a
 *                                                    head's digests are one contiguous
 *                                                    stream for the page scan
 *   page_table  [batch][max_pages]            int32  logical page -> physical page
 *   seq_lens    [batch]                       int32  tokens stored per sequence
 *   last_loaded [batch][h_k][max_pages]       int32  A of Alg. 2: last decode step in
 *                                                    which each logical page was
 *                                                    loaded; the caller initialises it
 *                                                    to -1 before the first step.
 * Slots beyond seq_lens are never read as keys; their values are zeroed before use. */
typedef struct retro_kv_cache {
  void* k_cache;
  void* v_cache;
  void* digest;
  const int32_t* page_table;
  int32_t* seq_lens;
  int32_t* last_loaded;
} retro_kv_cache;

/* Output of page selection (PageSelect + UpdateAndBuildMask).
 *   selected     [batch][h_k][k_max]  int32  logical page ids in ascending order,
 *                                            -1 after the first num_selected entries
 *   mask         [batch][h_k][k_max]  int32  M of Alg. 2: last_loaded of each selected
 *                                            page before this step (-1 padding)
 *   num_selected [batch][h_k]         int32
 * with k_max = retro_k_max(dims). */
typedef struct retro_selection {
  int32_t* selected;
  int32_t* mask;
  int32_t* num_selected;
} retro_selection;

/* The attention output cache (Sec. 2.3, "Attention Output Cache"): for each of the
 * last W steps tau, the output of tau's query merged over every supplement so
 * far, in ring slot tau mod W.
 *   o_cache   [batch][W][h_q][d]  fp32
 *   lse_cache [batch][W][h_q]     fp32 natural-log normaliser (log of alpha)
 * Slots are only read after the step that wrote them; no initialisation needed.
 * Both may be NULL when W == 0. */
typedef struct retro_output_cache {
  float* o_cache;
  float* lse_cache;
} retro_output_cache;

/* Library version string. */
const char* retro_version(void);

/* Human-readable name of a status code. */
const char* retro_status_string(int32_t status);

/* Validate dims; on success write k_max = min(budget_tokens / page_size, max_pages). */
retro_status retro_k_max(const retro_dims* dims, int32_t* k_max);

/* Bytes of scratch the select / attend / step calls need for these dims.  The
 * workspace holds, besides scratch, the words through which the workgroups of
 * one launch hand work to each other and a sticky error word: zero-fill it once
 * before its first use and let one call at a time use it (calls sharing a
 * workspace are ordered on one stream).  Use it with the dims it was sized for:
 * a one-launch step (see retro_step) on a workspace last used by a one-launch
 * step of another geometry sets the error word instead of running (its outputs
 * are NaN) until the workspace is zero-filled again. */
retro_status retro_workspace_size(const retro_dims* dims, size_t* bytes);

/* Bulk-store n_tokens tokens of sequence `seq` at positions start_pos ..
 * start_pos+n_tokens-1 (k_src, v_src: [n_tokens][h_k][d] dtype, device) and
 * rebuild the digests of the pages they touch.  start_pos must equal the
 * sequence's current seq_lens entry, which becomes start_pos + n_tokens.  For the
 * prefill that precedes the first decode step: last_loaded is not touched. */
retro_status retro_prefill_kv(const retro_dims* dims, const retro_kv_cache* cache, int32_t seq,
                              int32_t start_pos, int32_t n_tokens, const void* k_src,
                              const void* v_src, void* stream);

/* AppendKV (Alg. 1) of one token per sequence (k_new, v_new: [batch][h_k][d] dtype)
 * at position seq_lens[b], which is then incremented.  The page's digest widens to
 * the new key (or starts at it for the page's first slot), and last_loaded of that
 * page is set to step-1 for every head: Alg. 2's current-page rule, applied when a
 * page receives a key newer than every past query.  May be called several times
 * per step (several tokens per step).  A token whose logical page is not mapped
 * (page_table entry < 0 or >= num_phys_pages, or position >= max_pages*P) is
 * dropped and seq_lens is left unchanged. */
retro_status retro_append_kv(const retro_dims* dims, int32_t step, const retro_kv_cache* cache,
                             const void* k_new, const void* v_new, void* stream);

/* AppendKV (Alg. 1) of n_tokens tokens per sequence in order, with the result of
 * n_tokens calls of retro_append_kv (token j of sequence b at position
 * seq_lens[b] + j, digests widened, last_loaded of every page receiving a key set
 * to step-1 for every head), in one launch per 64 tokens: for steps that add
 * several tokens (e.g. the tokens before the last of a multi-token step, whose
 * last token goes through retro_step).  k_new / v_new [n_tokens][batch][h_k][d]
 * (dtype), device memory, read only.  The first token whose logical page is not
 * mapped (page_table entry < 0 or >= num_phys_pages, or position >= max_pages*P)
 * is dropped with every later token of the call, and seq_lens[b] advances by
 * the number appended.  n_tokens = 0 does nothing; n_tokens < 0 or a null
 * k_new / v_new (n_tokens > 0) is RETRO_EINVAL. */
retro_status retro_append_kv_tokens(const retro_dims* dims, int32_t step,
                                    const retro_kv_cache* cache, int32_t n_tokens,
                                    const void* k_new, const void* v_new, void* stream);

/* UpdateKV (Alg. 1; Sec. 3.3, retrospective KV cache update): the keys and values
 * of the n_tokens most recent stored tokens of every sequence b (positions
 * seq_lens[b] - n_tokens .. seq_lens[b] - 1; those below 0 are skipped) are
 * overwritten with k_upd / v_upd [batch][n_tokens][h_k][d] (dtype; row j is
 * position seq_lens[b] - n_tokens + j), e.g. re-embedded from the previous
 * layer's updated outputs, and the digest of every page they touch is recomputed
 * as the element-wise min / max over its stored keys.  Called before the step's
 * append (Alg. 1 order), with n_tokens = W for the window's past tokens.
 * last_loaded and seq_lens are unchanged.  n_tokens = 0 does nothing. */
retro_status retro_update_kv(const retro_dims* dims, const retro_kv_cache* cache,
                             int32_t n_tokens, const void* k_upd, const void* v_upd,
                             void* stream);

/* PageSelect + UpdateAndBuildMask (Alg. 1, Alg. 2) for the current query
 * q_cur [batch][h_q][d] (dtype).
 *   score of page p of KV head h = sum over the G query heads g of h of
 *     sum_i max(q_gi * Kmin_pi, q_gi * Kmax_pi)                  eq. (quest_score)
 *   evaluated in fp32: products rounded to fp32, the d terms summed as a perfect
 *   binary tree over index order, the G head sums added in order, then + 0.0f.
 *   The k = min(B_t/P, ceil(seq_len/P)) best pages by (score descending, page index
 *   ascending) are written in ascending order; then for each selected page p, in
 *   order: mask = last_loaded[p]; last_loaded[p] = step.
 * Page selection is exact: it depends on no floating-point reduction order other
 * than the one stated. */
/* (With dims->reuse_interval = f >= 2 and step mod f != 0 no score is computed:
 * the rows and counts `sel` holds are kept, and only the mask / last_loaded
 * loop above runs on them; q_cur is not read.) */
retro_status retro_select_pages(const retro_dims* dims, int32_t step, const void* q_cur,
                                const retro_kv_cache* cache, const retro_selection* sel,
                                void* workspace, size_t ws_bytes, void* stream);

/* Attention of the W+1 window queries q_window [batch][W+1][h_q][d] (dtype; row W
 * is step t) over the selected pages.  Row r (tau = t-W+r) uses page p iff tau >= 0
 * and (r == W or mask[p] < tau); every stored token of a used page counts.
 * Output per row and query head: o_part [batch][W+1][h_q][d] fp32 (softmax-weighted
 * values) and lse_part [batch][W+1][h_q] fp32 = ln sum exp(sm_scale * q.k);
 * an empty set gives (0, -inf).  Reads only; writes o_part, lse_part, workspace. */
retro_status retro_decode_attend(const retro_dims* dims, int32_t step, const void* q_window,
                                 const retro_kv_cache* cache, const retro_selection* sel,
                                 float* o_part, float* lse_part, void* workspace,
                                 size_t ws_bytes, void* stream);

/* The attention pass of retro_decode_attend alone, as one kernel launch: each
 * split's partial (O, LSE) stays in the workspace (library-private layout) and
 * nothing else is written.  Meant for timing the page-gather attention kernel in
 * isolation (the paper's kernel-level breakdown separates it from the merge);
 * callers wanting outputs use retro_decode_attend or retro_step. */
retro_status retro_decode_attend_partials(const retro_dims* dims, int32_t step,
                                          const void* q_window, const retro_kv_cache* cache,
                                          const retro_selection* sel, void* workspace,
                                          size_t ws_bytes, void* stream);

/* The kernel launch of retro_step that ends in the attention partials, alone:
 * page scores (eq. quest_score), selection (top-k + UpdateAndBuildMask's mask,
 * Alg. 2) and attention, with the sequence lengths of `cache` (no token is
 * appended).  Where retro_step scores in a launch of its own (see retro_step),
 * the launch starts from the page scores the last retro_step or
 * retro_select_pages call with this workspace left in it.  Writes the page
 * scores, sel's rows, mask and count (mask values from last_loaded as it
 * stands, which this call does not update) and the splits' partials in the
 * workspace.  Meant for timing the step's dominant kernel in isolation;
 * returns RETRO_EUNSUPPORTED where retro_step selects outside the attention
 * launch (max_pages > 6144). */
retro_status retro_step_attend_partials(const retro_dims* dims, int32_t step,
                                        const void* q_window, const retro_kv_cache* cache,
                                        const retro_selection* sel, void* workspace,
                                        size_t ws_bytes, void* stream);

/* The page scores, eq. (quest_score) in the fp32 order of retro_select_pages,
 * that the last retro_step, retro_step_attend_partials or retro_select_pages
 * call with this workspace computed: copied (asynchronously, on `stream`) to
 * scores [batch][h_k][max_pages] fp32, device memory.  Entries of pages at or
 * past a sequence's page count are unspecified.  Meant for checking the scores
 * bit for bit; workspace as sized by retro_workspace_size for these dims. */
retro_status retro_copy_scores(const retro_dims* dims, const void* workspace, size_t ws_bytes,
                               float* scores, void* stream);

/* MergeOutput + CacheOutput (Alg. 1; eq. merged_attn_general) for step t.
 * For each query head and row r with tau = t-W+r >= 0:
 *   r == W   : out = part; pushed to slot t mod W;
 *   0 < r < W: out = merge(slot tau mod W, part); written back to the slot;
 *   r == 0   : out = merge(slot, part) is final (the query leaves the window), and
 *              the slot (t-W) mod W = t mod W is then reused by row W;
 * where merge((O_a,Z_a),(O_b,Z_b)) = ((e^Za O_a + e^Zb O_b)/(e^Za + e^Zb),
 * ln(e^Za + e^Zb)), a -inf side contributing nothing.  Rows with tau < 0 give
 * o_out = 0, lse_out = -inf and touch no slot.
 *   o_out [batch][W+1][h_q][d] fp32, lse_out [batch][W+1][h_q] fp32. */
retro_status retro_merge_output_cache(const retro_dims* dims, int32_t step, const float* o_part,
                                      const float* lse_part, const retro_output_cache* ocache,
                                      float* o_out, float* lse_out, void* stream);

/* One whole step: retro_append_kv(k_new, v_new), retro_select_pages(row W of
 * q_window), retro_decode_attend, retro_merge_output_cache, with the same
 * semantics, without materialising o_part / lse_part.
 * One launch where every workgroup of it fits on the GPU at once (as the
 * occupancy of its kernel times the compute units tells; up to 4480 pages per
 * sequence and 160 per workgroup, (window + 1) * group <= 128 rows, at most 64
 * KV heads and 1024 workgroups):
 * page scores (with the append), selection, attention, combine + merge, the
 * last_loaded update and the seq_lens advance, the workgroups of a KV head
 * handing each other scores and partial results through tagged words in
 * `workspace` (each word carries the launch's epoch; no counters, no fences).
 * That needs every workgroup resident at once: work of other streams or
 * processes holding compute units delays it until they free them; a wait that
 * runs past its bound (tens of milliseconds) sets the sticky error word in
 * `workspace`: the outputs of that step and of every later step with this
 * workspace are then NaN, and the output cache, last_loaded and seq_lens are
 * left as they were, until the workspace is zero-filled again
 * (RETRO_FLAG_TEST_WAIT_TIMEOUT in dims->flags makes every such wait give up
 * at once, for tests of that path).
 * Otherwise, or with RETRO_FLAG_SEPARATE_SCORES, three launches: the scores
 * (with the append), then attention with every attention workgroup selecting
 * in front of it, then combine + merge; with RETRO_FLAG_SELECT_IN_SCORES, when
 * the attention launch has 64 or more workgroups per KV head (each of which
 * would repeat the selection), or for max_pages > 6144, the selection runs at
 * the end of the score launch (or in a launch of its own) instead.  Steps
 * that keep an earlier selection (top-k reuse, retro_dims.reuse_interval) run
 * the append, Alg. 2 on the kept rows, attention and combine + merge as four
 * launches. */
retro_status retro_step(const retro_dims* dims, int32_t step, const void* q_window,
                        const void* k_new, const void* v_new, const retro_kv_cache* cache,
                        const retro_selection* sel, const retro_output_cache* ocache,
                        float* o_out, float* lse_out, void* workspace, size_t ws_bytes,
                        void* stream);

/* The number of kernel launches retro_step makes for these dims on the current
 * device in a step that selects (1: scores, selection, attention and merge in
 * one launch; 3 or 4: see retro_step; a top-k reuse step always makes 4), in
 * *launches.  Host only: nothing is enqueued. */
retro_status retro_step_launches(const retro_dims* dims, int32_t* launches);

/* retro_step for callers that cannot allocate (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation): the same step and
 * results, with the workspace in a static device array of the library (64 MiB
 * per GPU, held until the process ends) instead of a caller's buffer; the
 * caller still passes every input and output.  No allocation is made.
 * Steps whose retro_workspace_size exceeds 64 MiB return RETRO_ESCRATCH.
 * Every call on a GPU shares that GPU's array, which keeps the last call's
 * contents: a call whose dims (flags aside) differ from the previous call's on
 * the device first clears the part it uses, with a kernel on `stream`; if that
 * stream is being captured the call returns RETRO_ESCRATCH instead (make the
 * first call of a geometry outside the capture).  Calls that overlap on one
 * GPU (other streams or host threads) race on the array.  After a wait that
 * gives up (see retro_step), later calls fail until the dims change. */
retro_status retro_step_noalloc(const retro_dims* dims, int32_t step, const void* q_window,
                                const void* k_new, const void* v_new,
                                const retro_kv_cache* cache, const retro_selection* sel,
                                const retro_output_cache* ocache, float* o_out,
                                float* lse_out, void* stream);

/* ---- Projections of the multi-layer decode with re-embedding (Sec. 3.3) --------
 * Every layer projects the W+1 window rows of every sequence (rows = batch*(W+1),
 * at most 112) to queries, keys and values, and its merged outputs back to the
 * model width; the past rows are re-embedded from the layer below's updated
 * outputs, their new keys and values then go to retro_update_kv.  With so few
 * rows the products are bound by reading the weights, which are therefore kept
 * pre-tiled for the matrix cores.  bf16 weights and inputs, fp32 accumulation,
 * bf16 results rounded to nearest even.  Every pointer is a device address,
 * 16-byte aligned; the caller owns every buffer. */

/* Tiles a weight w [k][n] bf16 (row-major, y = x . w) into w_packed (k*n bf16, a
 * separate buffer): element (i, j) goes to [j/16][i/32][(i%32)/8][j%16][i%8].
 * Weights that share an input (query, key and value) are packed as one [k][n]
 * matrix with their columns side by side.  k % 32 == 0 and n % 16 == 0, else
 * RETRO_EUNSUPPORTED. */
retro_status retro_pack_weight(const void* w, int32_t k, int32_t n, void* w_packed,
                               void* stream);

/* q = x . Wq, k_out = x . Wk, v = x . Wv for x [rows][k] bf16 and a packed
 * [k][n_q + 2 n_kv] weight whose columns are Wq's, then Wk's, then Wv's; outputs
 * bf16 [rows][n_q], [rows][n_kv], [rows][n_kv] (for the window rows of a
 * decoder: [batch][W+1][h_q][d] and [batch][W+1][h_k][d]).  Supported: 1 <= rows
 * <= 112, k % 1024 == 0, n_q % 16 == n_kv % 16 == 0 (else RETRO_EUNSUPPORTED);
 * rows == 0 does nothing. */
retro_status retro_project_qkv(const void* x, int32_t rows, int32_t k, const void* w_packed,
                               int32_t n_q, int32_t n_kv, void* q, void* k_out, void* v,
                               void* stream);

/* retro_project_qkv for the window rows of one decoder layer (rows = batch *
 * (W+1), x [batch][W+1][k] bf16, a packed [k][(h_q + 2 h_k) d] weight) with the
 * layer's UpdateKV folded in (Alg. 1; Sec. 3.3): q [batch][W+1][h_q][d] receives
 * every row's query; k_new, v_new [batch][h_k][d] the newest row's key and value
 * (for retro_step, which appends them); the keys and values of the n_update rows
 * before the newest overwrite the sequence's last n_update stored tokens, as
 * retro_update_kv would (positions seq_lens[b] - n_update .. seq_lens[b] - 1,
 * those below 0 skipped), and the digests of the pages they touch are
 * recomputed.  Call it before the step, whose append advances seq_lens.  bf16
 * dims only; 0 <= n_update <= W; rows <= 112, k % 1024 == 0 (else
 * RETRO_EUNSUPPORTED). */
retro_status retro_project_qkv_update(const retro_dims* dims, const retro_kv_cache* cache,
                                      const void* x, int32_t k, const void* w_packed,
                                      int32_t n_update, void* q, void* k_new, void* v_new,
                                      void* stream);

/* The output projection and the residual add: y = bf16(o) . Wo for o [rows][k]
 * fp32 (a decoder's merged outputs o_out, k = h_q * d) and a packed [k][n]
 * weight, rounded to bf16; then h[r][j] += y[r][j] in fp32 (h [rows][n], the
 * residual stream, updated in place) and x_next = bf16(h) [rows][n] (the next
 * layer's input).  Supported shapes as for retro_project_qkv. */
retro_status retro_project_out(const float* o, int32_t rows, int32_t k, const void* w_packed,
                               int32_t n, float* h, void* x_next, void* stream);

/* The projections of the multi-layer decode (Sec. 3.3) for fp32 stacks:
 * y = x . w (accumulate == 0) or y += x . w (accumulate != 0: the output
 * projection added into the residual stream in place) for x [rows][k] and w
 * [k][n] fp32 row-major (not packed), y [rows][n] fp32; x and y must not
 * overlap.  Each output element is one fp32 fused multiply-add chain over
 * i = 0 .. k-1 in order, so results repeat exactly from run to run.  rows == 0
 * does nothing; rows > 65535 or rows * n >= 2^31 is RETRO_EUNSUPPORTED. */
retro_status retro_project_f32(const float* x, int32_t rows, int32_t k, const float* w,
                               int32_t n, float* y, int32_t accumulate, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* RETRO_H */
