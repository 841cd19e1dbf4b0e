// C ABI entry points: argument validation, geometry and workspace sizing, and the
// launch sequences of each call.  Nothing here allocates device memory.
#include <math.h>

#include "internal.h"
#include "proj.h"

namespace retro {

int attend_min_waves(int dtype, int D);

namespace {

constexpr int kTargetWorkgroups = 256;   // attention workgroups aimed for per call
constexpr int kMaxChunksPerSplit = 32;   // pages per split <= 64 (LDS page list)
constexpr int kMaxWaves = 8;
constexpr int kMaxRtw = 2;

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

}  // namespace

retro_status make_geometry(const retro_dims* d, Geometry* g) {
  if (!d || !g) return RETRO_EINVAL;
  if (d->batch < 1 || d->num_kv_heads < 1 || d->group < 1 || d->head_dim < 1 ||
      d->page_size < 1 || d->budget_tokens < 1 || d->window < 0 || d->max_pages < 1 ||
      d->num_phys_pages < 1)
    return RETRO_EINVAL;
  if (d->dtype != RETRO_F32 && d->dtype != RETRO_BF16) return RETRO_EINVAL;
  if (!(d->sm_scale >= 0.f) || isinf(d->sm_scale)) return RETRO_EINVAL;
  if (d->head_dim != 64 && d->head_dim != 128) return RETRO_EUNSUPPORTED;
  if (d->page_size != 16 && d->page_size != 32) return RETRO_EUNSUPPORTED;
  if (d->group > 16 || d->window > 64) return RETRO_EUNSUPPORTED;
  if ((int64_t)(d->window + 1) * d->group > 1024) return RETRO_EUNSUPPORTED;
  if (d->budget_tokens < d->page_size) return RETRO_EINVAL;
  if (d->budget_permille < 0 || d->budget_permille > 1000) return RETRO_EINVAL;
  if (d->max_pages > 16384) return RETRO_EUNSUPPORTED;
  if (d->flags & ~(RETRO_FLAG_SEPARATE_SCORES | RETRO_FLAG_SELECT_IN_SCORES |
                   RETRO_FLAG_TEST_WAIT_TIMEOUT))
    return RETRO_EINVAL;
  if ((int64_t)d->batch * d->num_kv_heads > 65535) return RETRO_EUNSUPPORTED;

  Geometry x{};
  x.batch = d->batch;
  x.hk = d->num_kv_heads;
  x.G = d->group;
  x.hq = d->num_kv_heads * d->group;
  x.D = d->head_dim;
  x.P = d->page_size;
  x.budget = d->budget_tokens;
  x.W = d->window;
  x.R = (d->window + 1) * d->group;
  x.max_pages = d->max_pages;
  x.num_phys = d->num_phys_pages;
  x.dtype = d->dtype;
  x.elt = d->dtype == RETRO_BF16 ? 2 : 4;
  x.budget_permille = d->budget_permille;
  {
    // the largest budget of any step: that of a full page-table row
    int64_t bt = d->budget_tokens;
    if (d->budget_permille > 0)
      bt = std::max<int64_t>(bt, (int64_t)d->max_pages * d->page_size * d->budget_permille / 1000);
    x.k_max = (int)std::min<int64_t>(bt / d->page_size, d->max_pages);
  }
  x.sm_scale = d->sm_scale > 0.f ? d->sm_scale : 1.0f / sqrtf((float)d->head_dim);

  x.chunk_pages = 32 / x.P;
  x.chunks_max = (x.k_max + x.chunk_pages - 1) / x.chunk_pages;
  const int bh = x.batch * x.hk;
  const int want_splits = std::max(1, (kTargetWorkgroups + bh - 1) / bh);
  x.chunks_per_split =
      std::min(kMaxChunksPerSplit, std::max(1, (x.chunks_max + want_splits - 1) / want_splits));
  x.n_splits = (x.chunks_max + x.chunks_per_split - 1) / x.chunks_per_split;
  x.pages_per_split = x.chunks_per_split * x.chunk_pages;
  if (x.n_splits > 65535) return RETRO_EUNSUPPORTED;
  // one KV head's split partials are read through a 2 GiB buffer window
  if ((int64_t)x.n_splits * x.R * x.D * (int64_t)sizeof(float) >= (int64_t)1 << 31)
    return RETRO_EUNSUPPORTED;

  x.row_tiles = (x.R + 15) / 16;
  x.n_rgroups = (x.row_tiles + kMaxWaves * kMaxRtw - 1) / (kMaxWaves * kMaxRtw);
  x.tiles_per_group = (x.row_tiles + x.n_rgroups - 1) / x.n_rgroups;
  x.rtw = (x.tiles_per_group + kMaxWaves - 1) / kMaxWaves;
  // eight wavefronts whatever the number of row tiles: the idle ones still
  // share the staging of every chunk (0.2 us faster per attention launch at
  // the headline shape than one wavefront per tile)
  x.waves = std::max(std::max((x.tiles_per_group + x.rtw - 1) / x.rtw, attend_min_waves(x.dtype, x.D)),
                     kMaxWaves);
  if ((int64_t)x.hk * x.n_rgroups > 65535) return RETRO_EUNSUPPORTED;
  x.flags = d->flags;
  if (d->reuse_interval < 0) return RETRO_EINVAL;
  x.reuse = d->reuse_interval;

  const size_t bhs = (size_t)bh;
  // per workgroup of the one-launch step: launch count, geometry fingerprint
  // and failure mark, 128 B each; first in every geometry's layout, so that a
  // workspace last used with another geometry shows that geometry's
  // fingerprint in every line
  x.ws_heads = 0;
  size_t off = (size_t)kCtlLines * 128;
  x.ws_scores = off;
  off += align256(bhs * x.max_pages * sizeof(float));
  x.ws_phys = off;
  off += align256(bhs * x.k_max * sizeof(int32_t));
  x.ws_opart = off;
  off += align256(bhs * x.n_splits * x.R * x.D * sizeof(float));
  x.ws_lpart = off;
  off += align256(bhs * x.n_splits * x.R * sizeof(float));
  x.ws_err = off;  // sticky error word (a bounded wait ran out, or a foreign geometry)
  off += 256;
  x.ws_sel = off;  // per-head counters of the score + selection launch
  off += align256(bhs * kSelCounterInts * (1 + kSelMaxGroups) * sizeof(int32_t));
  x.ws_tok = off;  // per KV head: the step token's page when not kept (selection in attention)
  off += align256(bhs * sizeof(int32_t));
  x.ws_tagged = off;  // the one-launch step's tagged score words, then its key-range words
  off += align256(bhs * (x.max_pages + 2 * (size_t)x.n_splits * x.n_rgroups) * sizeof(uint64_t));
  x.ws_lse_tag = off;  // that step's tagged log-normalisers, [b * h_k][R][splits]
  off += align256(bhs * x.R * x.n_splits * sizeof(uint64_t));
  x.ws_head_tag = off;  // that step's per-head words (selection done)
  off += align256(bhs * sizeof(uint64_t));
  x.ws_dummy = off;  // never written: the stand-in of empty loads
  off += 256;
  x.ws_total = off;
  *g = x;
  return RETRO_OK;
}

}  // namespace retro

using retro::Geometry;

namespace {

retro_status from_hip(hipError_t e) { return e == hipSuccess ? RETRO_OK : RETRO_EHIP; }

bool cache_ok(const retro_kv_cache* c) {
  return c && c->k_cache && c->v_cache && c->digest && c->page_table && c->seq_lens &&
         c->last_loaded;
}

bool sel_ok(const retro_selection* s) { return s && s->selected && s->mask && s->num_selected; }

retro_status prepare(const retro_dims* dims, int32_t step, Geometry* g) {
  retro_status st = retro::make_geometry(dims, g);
  if (st != RETRO_OK) return st;
  if (step < 0) return RETRO_EINVAL;
  return RETRO_OK;
}

retro_status check_ws(const Geometry& g, void* ws, size_t ws_bytes) {
  if (!ws || ws_bytes < g.ws_total) return RETRO_EWORKSPACE;
  return RETRO_OK;
}

float* ws_at(void* ws, size_t off) { return reinterpret_cast<float*>((char*)ws + off); }

// retro_step's launch plan: scores, selection and attention in one launch
// where every workgroup of it fits on the GPU at once and the caller did not
// ask for a separate score launch
bool one_launch(const Geometry& g) {
  return !(g.flags & (RETRO_FLAG_SEPARATE_SCORES | RETRO_FLAG_SELECT_IN_SCORES)) &&
         retro::step_attend_supported(g);
}

// bounded waits: RETRO_FLAG_TEST_WAIT_TIMEOUT makes each give up after a few
// polls, its awaited tag being out of reach
int wait_limit(const Geometry& g) {
  return (g.flags & RETRO_FLAG_TEST_WAIT_TIMEOUT) ? 4 : retro::kSpinLimit;
}
uint32_t wait_bias(const Geometry& g) {
  return (g.flags & RETRO_FLAG_TEST_WAIT_TIMEOUT) ? 0x40000000u : 0u;
}

}  // namespace

extern "C" {

const char* retro_version(void) { return "retro-mi355x 0.1.0 (gfx950)"; }

const char* retro_status_string(int32_t status) {
  switch (status) {
    case RETRO_OK: return "RETRO_OK";
    case RETRO_EINVAL: return "RETRO_EINVAL: invalid argument";
    case RETRO_EUNSUPPORTED: return "RETRO_EUNSUPPORTED: shape outside the supported range";
    case RETRO_EHIP: return "RETRO_EHIP: HIP launch failed";
    case RETRO_EWORKSPACE: return "RETRO_EWORKSPACE: workspace missing or too small";
    case RETRO_ESCRATCH:
      return "RETRO_ESCRATCH: the step needs more than the static scratch, or its clear would be captured";
    default: return "unknown retro_status";
  }
}

retro_status retro_k_max(const retro_dims* dims, int32_t* k_max) {
  Geometry g;
  if (!k_max) return RETRO_EINVAL;
  retro_status st = retro::make_geometry(dims, &g);
  if (st != RETRO_OK) return st;
  *k_max = g.k_max;
  return RETRO_OK;
}

retro_status retro_workspace_size(const retro_dims* dims, size_t* bytes) {
  Geometry g;
  if (!bytes) return RETRO_EINVAL;
  retro_status st = retro::make_geometry(dims, &g);
  if (st != RETRO_OK) return st;
  *bytes = g.ws_total;
  return RETRO_OK;
}

retro_status retro_prefill_kv(const retro_dims* dims, const retro_kv_cache* cache, int32_t seq,
                              int32_t start_pos, int32_t n_tokens, const void* k_src,
                              const void* v_src, void* stream) {
  Geometry g;
  retro_status st = retro::make_geometry(dims, &g);
  if (st != RETRO_OK) return st;
  if (!cache_ok(cache) || !k_src || !v_src) return RETRO_EINVAL;
  if (seq < 0 || seq >= g.batch || start_pos < 0 || n_tokens < 0) return RETRO_EINVAL;
  if ((int64_t)start_pos + n_tokens > (int64_t)g.max_pages * g.P) return RETRO_EINVAL;
  return from_hip(retro::launch_prefill(g, *cache, seq, start_pos, n_tokens, k_src, v_src,
                                        (hipStream_t)stream));
}

retro_status retro_append_kv(const retro_dims* dims, int32_t step, const retro_kv_cache* cache,
                             const void* k_new, const void* v_new, void* stream) {
  Geometry g;
  retro_status st = prepare(dims, step, &g);
  if (st != RETRO_OK) return st;
  if (!cache_ok(cache) || !k_new || !v_new) return RETRO_EINVAL;
  return from_hip(retro::launch_append(g, step, *cache, k_new, v_new, (hipStream_t)stream));
}

retro_status retro_append_kv_tokens(const retro_dims* dims, int32_t step,
                                    const retro_kv_cache* cache, int32_t n_tokens,
                                    const void* k_new, const void* v_new, void* stream) {
  Geometry g;
  retro_status st = prepare(dims, step, &g);
  if (st != RETRO_OK) return st;
  if (!cache_ok(cache) || n_tokens < 0) return RETRO_EINVAL;
  if (n_tokens == 0) return RETRO_OK;
  if (!k_new || !v_new) return RETRO_EINVAL;
  return from_hip(retro::launch_append_tokens(g, step, *cache, n_tokens, k_new, v_new,
                                              (hipStream_t)stream));
}

retro_status retro_update_kv(const retro_dims* dims, const retro_kv_cache* cache,
                             int32_t n_tokens, const void* k_upd, const void* v_upd,
                             void* stream) {
  Geometry g;
  retro_status st = make_geometry(dims, &g);
  if (st != RETRO_OK) return st;
  if (!cache_ok(cache) || n_tokens < 0) return RETRO_EINVAL;
  if (n_tokens == 0) return RETRO_OK;
  if (!k_upd || !v_upd) return RETRO_EINVAL;
  if (n_tokens > g.max_pages * g.P) return RETRO_EINVAL;
  return from_hip(retro::launch_update_kv(g, *cache, n_tokens, k_upd, v_upd, (hipStream_t)stream));
}

retro_status retro_project_qkv_update(const retro_dims* dims, const retro_kv_cache* cache,
                                      const void* x, int32_t k, const void* w_packed,
                                      int32_t n_update, void* q, void* k_new, void* v_new,
                                      void* stream) {
  Geometry g;
  retro_status st = make_geometry(dims, &g);
  if (st != RETRO_OK) return st;
  if (!cache_ok(cache) || !x || !w_packed || !q || !k_new || !v_new || k <= 0 ||
      n_update < 0 || n_update > g.W)
    return RETRO_EINVAL;
  if ((reinterpret_cast<uintptr_t>(x) & 15u) || (reinterpret_cast<uintptr_t>(w_packed) & 15u))
    return RETRO_EINVAL;
  if (!retro::project_qkv_update_supported(g, k)) return RETRO_EUNSUPPORTED;
  return from_hip(retro::launch_project_qkv_update(g, *cache, x, k, w_packed, n_update, q, k_new,
                                                   v_new, (hipStream_t)stream));
}

retro_status retro_select_pages(const retro_dims* dims, int32_t step, const void* q_cur,
                                const retro_kv_cache* cache, const retro_selection* sel,
                                void* workspace, size_t ws_bytes, void* stream) {
  Geometry g;
  retro_status st = prepare(dims, step, &g);
  if (st != RETRO_OK) return st;
  if (!q_cur || !cache_ok(cache) || !sel_ok(sel)) return RETRO_EINVAL;
  if ((st = check_ws(g, workspace, ws_bytes)) != RETRO_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  if (retro::reuse_step(g, step))  // top-k reuse: Alg. 2 on the rows sel holds
    return from_hip(retro::launch_reuse_mask(g, step, *cache, *sel, s));
  float* scores = ws_at(workspace, g.ws_scores);
  int32_t* counters = reinterpret_cast<int32_t*>((char*)workspace + g.ws_sel);
  hipError_t e = retro::launch_score(g, step, q_cur, (int64_t)g.hq * g.D, *cache, nullptr, nullptr,
                                     scores, sel, nullptr, counters, s);
  if (e == hipSuccess && !retro::score_selects(g))
    e = retro::launch_topk_mask(g, step, scores, *cache, *sel, nullptr, s);
  return from_hip(e);
}

retro_status retro_decode_attend(const retro_dims* dims, int32_t step, const void* q_window,
                                 const retro_kv_cache* cache, const retro_selection* sel,
                                 float* o_part, float* lse_part, void* workspace,
                                 size_t ws_bytes, void* stream) {
  Geometry g;
  retro_status st = prepare(dims, step, &g);
  if (st != RETRO_OK) return st;
  if (!q_window || !cache_ok(cache) || !sel_ok(sel) || !o_part || !lse_part) return RETRO_EINVAL;
  if ((st = check_ws(g, workspace, ws_bytes)) != RETRO_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  float* o_ws = ws_at(workspace, g.ws_opart);
  float* l_ws = ws_at(workspace, g.ws_lpart);
  hipError_t e = retro::launch_attend(g, step, q_window, *cache, *sel, nullptr, o_ws, l_ws,
                                      (char*)workspace + g.ws_dummy, s);
  if (e == hipSuccess)
    e = retro::launch_combine_merge(g, step, 0, o_ws, l_ws, sel->num_selected, nullptr, nullptr,
                                    o_part, lse_part, nullptr, nullptr, nullptr, nullptr, s);
  return from_hip(e);
}

retro_status retro_decode_attend_partials(const retro_dims* dims, int32_t step,
                                          const void* q_window, const retro_kv_cache* cache,
                                          const retro_selection* sel, void* workspace,
                                          size_t ws_bytes, void* stream) {
  Geometry g;
  retro_status st = prepare(dims, step, &g);
  if (st != RETRO_OK) return st;
  if (!q_window || !cache_ok(cache) || !sel_ok(sel)) return RETRO_EINVAL;
  if ((st = check_ws(g, workspace, ws_bytes)) != RETRO_OK) return st;
  return from_hip(retro::launch_attend(g, step, q_window, *cache, *sel, nullptr,
                                       ws_at(workspace, g.ws_opart), ws_at(workspace, g.ws_lpart),
                                       (char*)workspace + g.ws_dummy, (hipStream_t)stream));
}

retro_status retro_step_attend_partials(const retro_dims* dims, int32_t step,
                                        const void* q_window, const retro_kv_cache* cache,
                                        const retro_selection* sel, void* workspace,
                                        size_t ws_bytes, void* stream) {
  Geometry g;
  retro_status st = prepare(dims, step, &g);
  if (st != RETRO_OK) return st;
  if (!q_window || !cache_ok(cache) || !sel_ok(sel)) return RETRO_EINVAL;
  if ((st = check_ws(g, workspace, ws_bytes)) != RETRO_OK) return st;
  if (!retro::attend_selects(g)) return RETRO_EUNSUPPORTED;
  int32_t* phys = reinterpret_cast<int32_t*>((char*)workspace + g.ws_phys);
  int32_t* tok = reinterpret_cast<int32_t*>((char*)workspace + g.ws_tok);
  if (one_launch(g)) {
    int32_t* err = reinterpret_cast<int32_t*>((char*)workspace + g.ws_err);
    return from_hip(retro::launch_step_attend(g, step, q_window, nullptr, nullptr, *cache, *sel,
                                              workspace, ws_at(workspace, g.ws_opart),
                                              ws_at(workspace, g.ws_lpart), tok, err,
                                              wait_limit(g), wait_bias(g), nullptr, nullptr,
                                              nullptr, (hipStream_t)stream));
  }
  return from_hip(retro::launch_attend_select(g, step, q_window, *cache, *sel, phys,
                                              ws_at(workspace, g.ws_scores),
                                              ws_at(workspace, g.ws_opart),
                                              ws_at(workspace, g.ws_lpart), tok,
                                              (char*)workspace + g.ws_dummy, (hipStream_t)stream));
}

namespace {
// Attention workgroups per KV head from which the selection runs once per head
// at the end of the score launch instead of in front of every attention
// workgroup, which repeats it once per workgroup.  Measured per layer-step:
// 64 per head (131K-token tables, W = 64: 32 splits x 2 row groups) 50.2 us
// in the score launch vs 52.4 in the attention launch; 16 per head (the
// long-generation workload) 115.2 vs 111.4; 2 per head (batch 16) 77.4 vs 63.8.
constexpr int kSelectInScoresFrom = 64;

bool select_in_attention(const Geometry& gp) {
  if (!retro::attend_selects(gp) || (gp.flags & RETRO_FLAG_SELECT_IN_SCORES)) return false;
  return !(retro::score_selects(gp) && gp.n_splits * gp.n_rgroups >= kSelectInScoresFrom);
}
}  // namespace

retro_status retro_step_launches(const retro_dims* dims, int32_t* launches) {
  Geometry g;
  if (!launches) return RETRO_EINVAL;
  retro_status st = retro::make_geometry(dims, &g);
  if (st != RETRO_OK) return st;
  Geometry gp = g;
  gp.token_pending = 1;
  if (one_launch(gp)) {
    *launches = 1;
  } else if (select_in_attention(gp)) {
    *launches = 3;
  } else {
    *launches = retro::score_selects(gp) ? 3 : 4;
  }
  return RETRO_OK;
}

retro_status retro_copy_scores(const retro_dims* dims, const void* workspace, size_t ws_bytes,
                               float* scores, void* stream) {
  Geometry g;
  retro_status st = retro::make_geometry(dims, &g);
  if (st != RETRO_OK) return st;
  if (!scores) return RETRO_EINVAL;
  if (!workspace || ws_bytes < g.ws_total) return RETRO_EWORKSPACE;
  const size_t n = (size_t)g.batch * g.hk * g.max_pages * sizeof(float);
  return from_hip(hipMemcpyAsync(scores, (const char*)workspace + g.ws_scores, n,
                                 hipMemcpyDeviceToDevice, (hipStream_t)stream));
}

retro_status retro_merge_output_cache(const retro_dims* dims, int32_t step, const float* o_part,
                                      const float* lse_part, const retro_output_cache* ocache,
                                      float* o_out, float* lse_out, void* stream) {
  Geometry g;
  retro_status st = prepare(dims, step, &g);
  if (st != RETRO_OK) return st;
  if (!o_part || !lse_part || !o_out || !lse_out) return RETRO_EINVAL;
  if (g.W > 0 && (!ocache || !ocache->o_cache || !ocache->lse_cache)) return RETRO_EINVAL;
  return from_hip(retro::launch_combine_merge(g, step, 1, nullptr, nullptr, nullptr, o_part,
                                              lse_part, nullptr, nullptr, ocache, o_out, lse_out,
                                              nullptr, (hipStream_t)stream));
}

}  // extern "C"

extern "C" {

retro_status retro_step(const retro_dims* dims, int32_t step, const void* q_window,
                        const void* k_new, const void* v_new, const retro_kv_cache* cache,
                        const retro_selection* sel, const retro_output_cache* ocache,
                        float* o_out, float* lse_out, void* workspace, size_t ws_bytes,
                        void* stream) {
  Geometry g;
  retro_status st = prepare(dims, step, &g);
  if (st != RETRO_OK) return st;
  if (!q_window || !k_new || !v_new || !cache_ok(cache) || !sel_ok(sel) || !o_out || !lse_out)
    return RETRO_EINVAL;
  if (g.W > 0 && (!ocache || !ocache->o_cache || !ocache->lse_cache)) return RETRO_EINVAL;
  if ((st = check_ws(g, workspace, ws_bytes)) != RETRO_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  float* scores = ws_at(workspace, g.ws_scores);
  float* o_ws = ws_at(workspace, g.ws_opart);
  float* l_ws = ws_at(workspace, g.ws_lpart);
  const int64_t qbs = (int64_t)(g.W + 1) * g.hq * g.D;
  const char* q_cur = (const char*)q_window + (int64_t)g.W * g.hq * g.D * g.elt;
  int32_t* phys = reinterpret_cast<int32_t*>((char*)workspace + g.ws_phys);
  int32_t* tok = reinterpret_cast<int32_t*>((char*)workspace + g.ws_tok);
  int32_t* err = reinterpret_cast<int32_t*>((char*)workspace + g.ws_err);
  const void* dummy = (char*)workspace + g.ws_dummy;
  if (retro::reuse_step(g, step)) {
    // top-k reuse: the token's append (with Alg. 2's current-page rule and the
    // seq_lens advance), Alg. 2 on the kept selection, attention, combine + merge
    hipError_t e = retro::launch_append(g, step, *cache, k_new, v_new, s);
    if (e == hipSuccess) e = retro::launch_reuse_mask(g, step, *cache, *sel, s);
    if (e == hipSuccess)
      e = retro::launch_attend(g, step, q_window, *cache, *sel, nullptr, o_ws, l_ws, dummy, s);
    if (e == hipSuccess)
      e = retro::launch_combine_merge(g, step, 2, o_ws, l_ws, sel->num_selected, nullptr,
                                      nullptr, nullptr, nullptr, ocache, o_out, lse_out, cache, s);
    return from_hip(e);
  }
  // the launches of this step append the token in their first launch and use
  // the length with it; the combine + merge launch advances seq_lens
  Geometry gp = g;
  gp.token_pending = 1;
  if (one_launch(gp)) {
    // scores (+ the token's append), selection, attention, combine + merge,
    // last_loaded update and seq_lens advance in one launch
    return from_hip(retro::launch_step_attend(gp, step, q_window, k_new, v_new, *cache, *sel,
                                              workspace, o_ws, l_ws, tok, err, wait_limit(g),
                                              wait_bias(g), ocache, o_out, lse_out, s));
  }
  if (select_in_attention(gp)) {
    // score (+ the token's append) -> attention with the selection in front ->
    // combine + merge (+ last_loaded update, + seq_lens advance)
    hipError_t e = retro::launch_score(gp, step, q_cur, qbs, *cache, k_new, v_new, scores,
                                       nullptr, nullptr, nullptr, s);
    if (e == hipSuccess)
      e = retro::launch_attend_select(gp, step, q_window, *cache, *sel, phys, scores, o_ws, l_ws,
                                      tok, dummy, s);
    if (e == hipSuccess)
      e = retro::launch_combine_merge(gp, step, 2, o_ws, l_ws, sel->num_selected, nullptr,
                                      nullptr, nullptr, nullptr, ocache, o_out, lse_out, cache, s,
                                      sel->selected, tok);
    return from_hip(e);
  }
  // score (+ the token's append, + top-k + mask) -> [top-k + mask] -> attention
  // -> combine + merge (+ seq_lens advance)
  int32_t* counters = reinterpret_cast<int32_t*>((char*)workspace + g.ws_sel);
  hipError_t e = retro::launch_score(gp, step, q_cur, qbs, *cache, k_new, v_new, scores, sel, phys,
                                     counters, s);
  if (e == hipSuccess && !retro::score_selects(gp))
    e = retro::launch_topk_mask(gp, step, scores, *cache, *sel, phys, s);
  if (e == hipSuccess)
    e = retro::launch_attend(gp, step, q_window, *cache, *sel, phys, o_ws, l_ws, dummy, s);
  if (e == hipSuccess)
    e = retro::launch_combine_merge(gp, step, 2, o_ws, l_ws, sel->num_selected, nullptr, nullptr,
                                    nullptr, nullptr, ocache, o_out, lse_out, cache, s);
  return from_hip(e);
}

}  // extern "C"
