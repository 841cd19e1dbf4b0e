/*
 * CPU ORACLE for one decode step of retrospective sparse attention
 * ("Retrospective Sparse Attention for Efficient Long-Context Generation").
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may load, call or
 * link this file; only the test-suite, the smoke entry point and the CPU
 * baseline leg of the benchmark do.  It shares no code, header, table or
 * helper with the GPU library.
 *
 * It is deliberately plain and slow:
 *   - page digests: element-wise key min / max per page (Sec. 2.1, Quest);
 *   - page score:   eq. (quest_score), evaluated in fp32 in one fixed order
 *                   (see oracle_score) so that a selection is reproducible;
 *   - page select:  the k best pages, ties to the lower page index;
 *   - mask:         Alg. 2 (UpdateAndBuildMask), with its current-page rule applied
 *                   to every page written during the step (oracle_append);
 *   - attention:    eq. (update-org) for the current query and
 *                   eq. (update-sup) for the past queries of the window,
 *                   in fp64, two passes, no blocking;
 *   - merge:        eq. (merged_attn) / (merged_attn_general) written with
 *                   log-sum-exp normalisers, and the output cache push /
 *                   update / pop of Sec. 2.3 ("Attention Output Cache").
 *
 * Compile with  gcc -O2 -fopenmp -ffp-contract=off  (no -ffast-math): the
 * fp32 score order below must not be contracted or re-associated.
 *
 * Conventions (all arrays are caller-owned host memory, row-major):
 *   K, V        [batch][h_k][max_tokens][d]   float (values of the inputs)
 *   kmin, kmax  [batch][h_k][max_pages][d]    float
 *   A           [batch][h_k][max_pages]       int32, starts at -1
 *   seq_lens    [batch]                       int32, tokens stored
 *   q_window    [batch][W+1][h_q][d]          float, row W = step t
 *   o_cache     [batch][W][h_q][d]            double, slot = tau mod W
 *   lse_cache   [batch][W][h_q]               double
 *   selected, M [batch][h_k][k_max]           int32 (ascending page ids)
 *   o_part/out  [batch][W+1][h_q][d]          double
 *   lse_*       [batch][W+1][h_q]             double (natural log)
 * with h_q = h_k * group, max_pages = ceil(max_tokens / P) and
 * k_max = min(B_max / P, max_pages), B_max the budget of a sequence of
 * max_pages * P tokens (see budget_tokens_at).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
  int32_t batch;
  int32_t num_kv_heads;
  int32_t group;
  int32_t head_dim;
  int32_t page_size;
  int32_t budget;
  int32_t window;
  int32_t max_tokens;
  double sm_scale;
  int32_t budget_permille; /* relative budget in thousandths; 0: the fixed budget */
} oracle_dims;

static int64_t max_pages_of(const oracle_dims* g) {
  return (g->max_tokens + g->page_size - 1) / g->page_size;
}

/* The token budget of a step whose sequence holds len tokens (the step's own
 * token included): the fixed budget B, or with a relative budget (Sec. 4,
 * ablation; the setting of Table 1) len times the fraction, rounded down, but
 * at least B. */
static int64_t budget_tokens_at(const oracle_dims* g, int64_t len) {
  int64_t b = g->budget;
  if (g->budget_permille > 0) {
    const int64_t rel = len * g->budget_permille / 1000;
    if (rel > b) b = rel;
  }
  return b;
}

int32_t oracle_k_max(const oracle_dims* g) {
  int64_t mp = max_pages_of(g);
  int64_t k = budget_tokens_at(g, mp * g->page_size) / g->page_size;
  return (int32_t)(k < mp ? k : mp);
}

/* ---------------------------------------------------------------------------
 * Storage.  Appending token `pos` writes K/V and keeps the page digest equal to
 * the element-wise min / max over the page's stored keys: the first token of a
 * page initialises it, later tokens widen it.
 * ------------------------------------------------------------------------- */
static void store_token(const oracle_dims* g, int b, int pos, float* K, float* V,
                        float* kmin, float* kmax, const float* k_tok, const float* v_tok) {
  const int hk = g->num_kv_heads, d = g->head_dim, P = g->page_size;
  const int64_t mp = max_pages_of(g);
  const int page = pos / P;
  for (int h = 0; h < hk; ++h) {
    float* kd = K + (((int64_t)b * hk + h) * g->max_tokens + pos) * d;
    float* vd = V + (((int64_t)b * hk + h) * g->max_tokens + pos) * d;
    float* lo = kmin + (((int64_t)b * hk + h) * mp + page) * d;
    float* hi = kmax + (((int64_t)b * hk + h) * mp + page) * d;
    const float* ks = k_tok + (int64_t)h * d;
    const float* vs = v_tok + (int64_t)h * d;
    for (int i = 0; i < d; ++i) {
      kd[i] = ks[i];
      vd[i] = vs[i];
      if (pos % P == 0) {
        lo[i] = ks[i];
        hi[i] = ks[i];
      } else {
        if (ks[i] < lo[i]) lo[i] = ks[i];
        if (ks[i] > hi[i]) hi[i] = ks[i];
      }
    }
  }
}

/* Bulk prefill of sequence b with n tokens ([n][h_k][d]).  Prefill precedes the
 * first decode step, so the retrospective mask A is left untouched. */
int oracle_prefill(const oracle_dims* g, int32_t b, int32_t n, int32_t* seq_lens, float* K,
                   float* V, float* kmin, float* kmax, const float* k_src, const float* v_src) {
  const int64_t tok = (int64_t)g->num_kv_heads * g->head_dim;
  if (seq_lens[b] + n > g->max_tokens) return -1;
  for (int32_t j = 0; j < n; ++j) {
    store_token(g, b, seq_lens[b], K, V, kmin, kmax, k_src + j * tok, v_src + j * tok);
    seq_lens[b] += 1;
  }
  return 0;
}

/* AppendKV (Alg. 1) for one token per sequence (k_new, v_new: [batch][h_k][d]).
 * The page that receives the token then holds a key newer than every past query
 * of the window, so Alg. 2's current-page rule, A[p_curr] <- t - 1, is applied to it
 * here, at the moment it is written (for every head).  When a step appends
 * several tokens each written page gets the same treatment, which is what keeps
 * past queries away from any page holding a key newer than themselves. */
int oracle_append(const oracle_dims* g, int32_t step, int32_t* seq_lens, float* K, float* V,
                  float* kmin, float* kmax, int32_t* A, const float* k_new, const float* v_new) {
  const int hk = g->num_kv_heads;
  const int64_t tok = (int64_t)hk * g->head_dim;
  const int64_t mp = max_pages_of(g);
  for (int b = 0; b < g->batch; ++b)
    if (seq_lens[b] >= g->max_tokens) return -1;
  for (int b = 0; b < g->batch; ++b) {
    const int pos = seq_lens[b];
    store_token(g, b, pos, K, V, kmin, kmax, k_new + b * tok, v_new + b * tok);
    seq_lens[b] = pos + 1;
    for (int h = 0; h < hk; ++h) A[((int64_t)b * hk + h) * mp + pos / g->page_size] = step - 1;
  }
  return 0;
}

/* ---------------------------------------------------------------------------
 * UpdateKV (Alg. 1; Sec. 3.3, retrospective KV cache update): the keys and
 * values of the n most recent stored tokens of every sequence b (positions
 * seq_lens[b] - n .. seq_lens[b] - 1, those below 0 skipped) are replaced by
 * k_upd / v_upd ([batch][n][h_k][d], row j = position seq_lens[b] - n + j),
 * and the digest of every page holding one of them becomes the element-wise
 * min / max over all of that page's stored keys again.
 * ------------------------------------------------------------------------- */
void oracle_update_kv(const oracle_dims* g, int32_t n, const int32_t* seq_lens, float* K,
                      float* V, float* kmin, float* kmax, const float* k_upd,
                      const float* v_upd) {
  const int hk = g->num_kv_heads, d = g->head_dim, P = g->page_size;
  const int64_t mp = max_pages_of(g);
  for (int b = 0; b < g->batch; ++b) {
    const int len = seq_lens[b];
    const int first = len - n;
    for (int pos = first < 0 ? 0 : first; pos < len; ++pos)
      for (int h = 0; h < hk; ++h)
        for (int i = 0; i < d; ++i) {
          const int64_t src = (((int64_t)b * n + (pos - first)) * hk + h) * d + i;
          const int64_t dst = (((int64_t)b * hk + h) * g->max_tokens + pos) * d + i;
          K[dst] = k_upd[src];
          V[dst] = v_upd[src];
        }
    if (len <= 0 || n <= 0) continue;
    const int p0 = (first < 0 ? 0 : first) / P, p1 = (len - 1) / P;
    for (int page = p0; page <= p1; ++page)
      for (int h = 0; h < hk; ++h)
        for (int i = 0; i < d; ++i) {
          float lo = 0.f, hi = 0.f;
          for (int pos = page * P; pos < (page + 1) * P && pos < len; ++pos) {
            const float x = K[(((int64_t)b * hk + h) * g->max_tokens + pos) * d + i];
            if (pos == page * P || x < lo) lo = x;
            if (pos == page * P || x > hi) hi = x;
          }
          kmin[(((int64_t)b * hk + h) * mp + page) * d + i] = lo;
          kmax[(((int64_t)b * hk + h) * mp + page) * d + i] = hi;
        }
  }
}

/* ---------------------------------------------------------------------------
 * Page score, eq. (quest_score): score_j(Q) = sum_i max(Q_i Kmin_i, Q_i Kmax_i).
 * A KV head's page is scored for the sum over the query heads of its group
 * (page selection is per KV head, Sec. "Retrospective Mask").
 *
 * The paper's score is real-valued; to make a selection reproducible bit for
 * bit it is evaluated in fp32 in this fixed order:
 *   p_i  = max(fl(q_i * kmin_i), fl(q_i * kmax_i))
 *   s_g  = pairwise sum of p_0 .. p_{d-1}: a perfect binary tree whose leaves
 *          are the d terms in index order (d is a power of two);
 *   S    = ((s_0 + s_1) + s_2) + ... over the group's heads in order;
 *   score = S + 0.0f   (so a zero score is always +0).
 * ------------------------------------------------------------------------- */
static float pairwise_sum(float* t, int n) {
  for (int w = 1; w < n; w *= 2)
    for (int i = 0; i + w < n; i += 2 * w) t[i] = t[i] + t[i + w];
  return t[0];
}

void oracle_score(const oracle_dims* g, const float* q_cur, const float* kmin,
                  const float* kmax, const int32_t* seq_lens, float* scores) {
  const int hk = g->num_kv_heads, G = g->group, d = g->head_dim, P = g->page_size;
  const int64_t mp = max_pages_of(g);
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int b = 0; b < g->batch; ++b) {
    for (int h = 0; h < hk; ++h) {
      float* t = (float*)malloc(sizeof(float) * d);
      const int n = (seq_lens[b] + P - 1) / P;
      for (int p = 0; p < n; ++p) {
        const float* lo = kmin + (((int64_t)b * hk + h) * mp + p) * d;
        const float* hi = kmax + (((int64_t)b * hk + h) * mp + p) * d;
        float S = 0.0f;
        for (int gq = 0; gq < G; ++gq) {
          const float* q = q_cur + ((int64_t)b * hk * G + (int64_t)h * G + gq) * d;
          for (int i = 0; i < d; ++i) {
            const float a = q[i] * lo[i];
            const float c = q[i] * hi[i];
            t[i] = a > c ? a : c;
          }
          const float s = pairwise_sum(t, d);
          S = (gq == 0) ? s : S + s;
        }
        scores[((int64_t)b * hk + h) * mp + p] = S + 0.0f;
      }
      free(t);
    }
  }
}

/* ---------------------------------------------------------------------------
 * PageSelect (Alg. 1): keep the k = min(B_t / P, n_pages) best pages of the
 * current query, ordered by (score descending, page index ascending); emit them
 * in ascending page order, padding the row with -1.
 * ------------------------------------------------------------------------- */
typedef struct {
  float s;
  int32_t p;
} scored_page;

static int by_score_then_index(const void* x, const void* y) {
  const scored_page* a = (const scored_page*)x;
  const scored_page* b = (const scored_page*)y;
  if (a->s > b->s) return -1;
  if (a->s < b->s) return 1;
  return (a->p > b->p) - (a->p < b->p);
}

static int by_index(const void* x, const void* y) {
  const int32_t a = *(const int32_t*)x, b = *(const int32_t*)y;
  return (a > b) - (a < b);
}

void oracle_select(const oracle_dims* g, const float* scores, const int32_t* seq_lens,
                   int32_t* selected, int32_t* num_selected) {
  const int hk = g->num_kv_heads, P = g->page_size;
  const int64_t mp = max_pages_of(g);
  const int32_t kmax = oracle_k_max(g);
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int b = 0; b < g->batch; ++b) {
    for (int h = 0; h < hk; ++h) {
      const int n = (seq_lens[b] + P - 1) / P;
      const int64_t kb = budget_tokens_at(g, seq_lens[b]) / P;
      int k = kb < n ? (int)kb : n;
      if (k > kmax) k = kmax;
      scored_page* all = (scored_page*)malloc(sizeof(scored_page) * (n > 0 ? n : 1));
      for (int p = 0; p < n; ++p) {
        all[p].s = scores[((int64_t)b * hk + h) * mp + p];
        all[p].p = p;
      }
      qsort(all, n, sizeof(scored_page), by_score_then_index);
      int32_t* row = selected + ((int64_t)b * hk + h) * kmax;
      for (int i = 0; i < k; ++i) row[i] = all[i].p;
      qsort(row, k, sizeof(int32_t), by_index);
      for (int i = k; i < kmax; ++i) row[i] = -1;
      num_selected[b * hk + h] = k;
      free(all);
    }
  }
}

/* ---------------------------------------------------------------------------
 * UpdateAndBuildMask (Alg. 2), one KV head at a time: for every selected page,
 * in order, M gets the step in which the page was last loaded and A records the
 * current step.  (Its current-page rule, the override of the current page, happens at
 * append time, see oracle_append.)  Padding entries of M are -1.
 * ------------------------------------------------------------------------- */
void oracle_build_mask(const oracle_dims* g, int32_t step, const int32_t* selected,
                       const int32_t* num_selected, int32_t* A, int32_t* M) {
  const int hk = g->num_kv_heads;
  const int64_t mp = max_pages_of(g);
  const int32_t kmax = oracle_k_max(g);
  for (int b = 0; b < g->batch; ++b) {
    for (int h = 0; h < hk; ++h) {
      const int32_t* row = selected + ((int64_t)b * hk + h) * kmax;
      int32_t* m = M + ((int64_t)b * hk + h) * kmax;
      int32_t* a = A + ((int64_t)b * hk + h) * mp;
      const int k = num_selected[b * hk + h];
      for (int i = 0; i < k; ++i) {
        m[i] = a[row[i]];
        a[row[i]] = step;
      }
      for (int i = k; i < kmax; ++i) m[i] = -1;
    }
  }
}

/* ---------------------------------------------------------------------------
 * Attention over the window's W+1 queries.  Row r is the query of step
 * tau = t - W + r (row W is the current query).  Rows with tau < 0 do not exist
 * yet: (O, Z) = (0, -inf).  The current query attends every stored token of the
 * selected pages (eq. update-org).  A past query attends the selected pages it
 * has not seen, i.e. those whose mask value M (last step the page was loaded,
 * or the override of Alg. 2) is older than tau (eq. update-sup with the
 * masking rule of Sec. "Retrospective Mask").  Z is the natural-log sum of
 * exp(sm_scale * q.k) over the attended tokens; O the softmax-weighted values;
 * an empty set gives (0, -inf).
 * ------------------------------------------------------------------------- */
void oracle_attend(const oracle_dims* g, int32_t step, const float* q_window, const float* K,
                   const float* V, const int32_t* seq_lens, const int32_t* selected,
                   const int32_t* num_selected, const int32_t* M, double* o_part,
                   double* lse_part) {
  const int hk = g->num_kv_heads, G = g->group, d = g->head_dim, P = g->page_size;
  const int W = g->window, hq = hk * G;
  const int32_t kmax = oracle_k_max(g);
  const int rows = W + 1;
#pragma omp parallel for collapse(3) schedule(dynamic)
  for (int b = 0; b < g->batch; ++b) {
    for (int r = 0; r < rows; ++r) {
      for (int qh = 0; qh < hq; ++qh) {
        const int h = qh / G;
        const int tau = step - W + r;
        double* o = o_part + (((int64_t)b * rows + r) * hq + qh) * d;
        double* z = lse_part + ((int64_t)b * rows + r) * hq + qh;
        for (int i = 0; i < d; ++i) o[i] = 0.0;
        *z = -INFINITY;
        if (tau < 0) continue;
        const float* q = q_window + (((int64_t)b * rows + r) * hq + qh) * d;
        const int32_t* sel = selected + ((int64_t)b * hk + h) * kmax;
        const int32_t* m = M + ((int64_t)b * hk + h) * kmax;
        const int k = num_selected[b * hk + h];
        const int L = seq_lens[b];
        double* s = (double*)malloc(sizeof(double) * ((int64_t)k * P + 1));
        int32_t* tok = (int32_t*)malloc(sizeof(int32_t) * ((int64_t)k * P + 1));
        int n = 0;
        for (int j = 0; j < k; ++j) {
          if (!(r == W || m[j] < tau)) continue;
          const int p = sel[j];
          for (int pos = p * P; pos < (p + 1) * P && pos < L; ++pos) {
            const float* kk = K + (((int64_t)b * hk + h) * g->max_tokens + pos) * d;
            double acc = 0.0;
            for (int i = 0; i < d; ++i) acc += (double)q[i] * (double)kk[i];
            s[n] = g->sm_scale * acc;
            tok[n] = pos;
            ++n;
          }
        }
        if (n > 0) {
          double mx = s[0];
          for (int e = 1; e < n; ++e)
            if (s[e] > mx) mx = s[e];
          double sum = 0.0;
          for (int e = 0; e < n; ++e) sum += exp(s[e] - mx);
          for (int e = 0; e < n; ++e) {
            const double w = exp(s[e] - mx) / sum;
            const float* vv = V + (((int64_t)b * hk + h) * g->max_tokens + tok[e]) * d;
            for (int i = 0; i < d; ++i) o[i] += w * (double)vv[i];
          }
          *z = mx + log(sum);
        }
        free(s);
        free(tok);
      }
    }
  }
}

/* ---------------------------------------------------------------------------
 * MergeOutput + CacheOutput (Alg. 1) with eq. (merged_attn_general): a cached
 * output (O_a, normaliser alpha_a = e^{Z_a}) and a supplementary output
 * (O_b, alpha_b = e^{Z_b}) combine to
 *     O = (alpha_a O_a + alpha_b O_b) / (alpha_a + alpha_b),
 *     alpha = alpha_a + alpha_b   i.e.   Z = log(e^{Z_a} + e^{Z_b}),
 * evaluated relative to max(Z_a, Z_b); a side with Z = -inf contributes nothing
 * and two empty sides give (0, -inf).
 * ------------------------------------------------------------------------- */
static void lse_merge(int d, const double* oa, double za, const double* ob, double zb,
                      double* o, double* z) {
  const double m = za > zb ? za : zb;
  if (m == -INFINITY) {
    for (int i = 0; i < d; ++i) o[i] = 0.0;
    *z = -INFINITY;
    return;
  }
  const double wa = exp(za - m), wb = exp(zb - m);
  for (int i = 0; i < d; ++i) o[i] = (wa * oa[i] + wb * ob[i]) / (wa + wb);
  *z = m + log(wa + wb);
}

/* The cache holds, for each of the last W steps tau, the output of tau's query
 * merged over every supplement so far, in slot tau mod W.  For each active row:
 *   row W (tau = t)         : output = the current attention; pushed to slot t mod W;
 *   rows 0 < r < W          : merged with their slot, written back (Update);
 *   row 0 (tau = t - W)     : merged with its slot and returned as final; its slot
 *                             (t - W) mod W = t mod W is then reused (Pop, then Push).
 * Rows with tau < 0 give (0, -inf) and touch no slot. */
void oracle_merge(const oracle_dims* g, int32_t step, const double* o_part,
                  const double* lse_part, double* o_cache, double* lse_cache, double* o_out,
                  double* lse_out) {
  const int hq = g->num_kv_heads * g->group, d = g->head_dim, W = g->window;
  const int rows = W + 1;
  double* tmp = (double*)malloc(sizeof(double) * d);
  for (int b = 0; b < g->batch; ++b) {
    for (int qh = 0; qh < hq; ++qh) {
      for (int r = 0; r < rows; ++r) {
        const int tau = step - W + r;
        const double* op = o_part + (((int64_t)b * rows + r) * hq + qh) * d;
        const double zp = lse_part[((int64_t)b * rows + r) * hq + qh];
        double* oo = o_out + (((int64_t)b * rows + r) * hq + qh) * d;
        double* zo = lse_out + ((int64_t)b * rows + r) * hq + qh;
        if (tau < 0) {
          for (int i = 0; i < d; ++i) oo[i] = 0.0;
          *zo = -INFINITY;
          continue;
        }
        if (r == W) {
          for (int i = 0; i < d; ++i) oo[i] = op[i];
          *zo = zp;
          continue;
        }
        const int slot = tau % W;
        double* oc = o_cache + (((int64_t)b * W + slot) * hq + qh) * d;
        double* zc = lse_cache + ((int64_t)b * W + slot) * hq + qh;
        double z;
        lse_merge(d, oc, *zc, op, zp, tmp, &z);
        for (int i = 0; i < d; ++i) oo[i] = tmp[i];
        *zo = z;
        if (r > 0) {
          for (int i = 0; i < d; ++i) oc[i] = tmp[i];
          *zc = z;
        }
      }
      if (W > 0) {
        const int slot = step % W;
        const double* op = o_part + (((int64_t)b * rows + W) * hq + qh) * d;
        double* oc = o_cache + (((int64_t)b * W + slot) * hq + qh) * d;
        for (int i = 0; i < d; ++i) oc[i] = op[i];
        lse_cache[((int64_t)b * W + slot) * hq + qh] = lse_part[((int64_t)b * rows + W) * hq + qh];
      }
    }
  }
  free(tmp);
}

/* Stand-alone LSE merge of two partial outputs (exposed for the merge pins). */
void oracle_lse_merge(int32_t d, const double* oa, double za, const double* ob, double zb,
                      double* o, double* z) {
  lse_merge(d, oa, za, ob, zb, o, z);
}

/* Threads the parallel loops above use (for reporting the CPU baseline). */
#ifdef _OPENMP
#include <omp.h>
#endif
int32_t oracle_num_threads(void) {
#ifdef _OPENMP
  return (int32_t)omp_get_max_threads();
#else
  return 1;
#endif
}
