// Private declarations shared by the library's HIP translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <algorithm>
#include <type_traits>

#include "retro.h"

namespace retro {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// bf16 values are carried as raw 16-bit patterns outside the MFMA code.
struct bf16_t {
  uint16_t bits;
};

// Workgroups are dispatched to the 8 XCDs round-robin.  Renumber them so that
// consecutive work units land on one XCD: unit u of n goes to XCD u / (n / 8).
// (Identity when n is not a multiple of 8.)
__device__ __forceinline__ int xcd_remap(int i, int n) {
  if (n % 8 != 0) return i;
  return (i % 8) * (n / 8) + i / 8;
}

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16_t x) {
  return __uint_as_float(static_cast<uint32_t>(x.bits) << 16);
}

// Validated, derived dimensions of one call.
struct Geometry {
  int batch, hk, G, hq, D, P, budget, W, R, max_pages, num_phys, dtype, elt;
  int k_max;          // selection row length
  int budget_permille;  // relative budget (0: the fixed budget B only)
  float sm_scale;     // resolved (never 0)
  // attention split geometry
  int chunk_pages;    // pages per 32-token chunk (2 for P=16, 1 for P=32)
  int chunks_max;     // chunks needed for k_max pages
  int chunks_per_split;
  int n_splits;       // splits per (b, h_k)
  int pages_per_split;
  int row_tiles;      // ceil(R / 16)
  int n_rgroups;      // row groups (workgroups sharing a split's pages)
  int tiles_per_group;
  int rtw;            // row tiles per wave
  int waves;          // waves per attention workgroup
  int flags;          // retro_dims.flags (RETRO_FLAG_*)
  int reuse;          // retro_dims.reuse_interval (top-k reuse; < 2: every step selects)
  // workspace layout (bytes): page scores, physical ids of the selection,
  // split partials, the sticky error word, the score launch's counters, the
  // step token's page per head, the one-launch step's tagged score words and
  // per-workgroup counter lines, its tagged log-normalisers of the partials and
  // per-head words, a dummy line (never written) for empty loads
  size_t ws_scores, ws_phys, ws_opart, ws_lpart, ws_err, ws_sel, ws_tok, ws_tagged, ws_heads,
      ws_lse_tag, ws_head_tag, ws_dummy, ws_total;
  // set for the launches of a step whose token is written by its score launch:
  // seq_lens does not count the token yet (the merge launch advances it), and
  // every launch uses the length with the token
  int token_pending;
};

// counters of the score + selection launch: per KV head 1 + kSelMaxGroups
// counters, each kSelCounterInts apart (one 128-byte line)
constexpr int kSelCounterInts = 32;
constexpr int kSelMaxGroups = 8;
// polls of a bounded wait (about 0.2 us each) before it gives up
constexpr int kSpinLimit = 1 << 18;
// control lines of the one-launch step (its largest grid)
constexpr int kCtlLines = 1024;

retro_status make_geometry(const retro_dims* d, Geometry* g);
int attend_min_waves(int dtype, int D);

// ---- launchers (return hipSuccess or the launch error) ----
hipError_t launch_append(const Geometry& g, int step, const retro_kv_cache& c, const void* k_new,
                         const void* v_new, hipStream_t s);
// n_tok tokens per sequence, k_new / v_new [n_tok][batch][h_k][d], in order
hipError_t launch_append_tokens(const Geometry& g, int step, const retro_kv_cache& c, int n_tok,
                                const void* k_new, const void* v_new, hipStream_t s);
hipError_t launch_prefill(const Geometry& g, const retro_kv_cache& c, int seq, int start, int n,
                          const void* k_src, const void* v_src, hipStream_t s);
// UpdateKV: the n most recent stored tokens of every sequence get new keys and
// values (k_upd, v_upd: [batch][n][h_k][d]); their pages' digests are recomputed.
hipError_t launch_update_kv(const Geometry& g, const retro_kv_cache& c, int n, const void* k_upd,
                            const void* v_upd, hipStream_t s);
// With g.token_pending, the score launch also appends the step's token
// (k_new, v_new: [batch][h_k][d]) as AppendKV does, without advancing seq_lens.
// With a selection, counters ([batch * h_k] ints of the workspace, zero
// between launches) and score_selects(g), it also runs top-k + mask (the last
// workgroup of each KV head); otherwise launch_topk_mask must follow.
bool score_selects(const Geometry& g);
hipError_t launch_score(const Geometry& g, int step, const void* q_cur, int64_t q_batch_stride,
                        const retro_kv_cache& c, const void* k_new, const void* v_new,
                        float* scores, const retro_selection* sel, int32_t* sel_phys,
                        int32_t* counters, hipStream_t s);
// Top-k reuse steps: UpdateAndBuildMask (Alg. 2) on the rows `sel` holds (mask
// values from last_loaded, then last_loaded = step for the kept pages).
bool reuse_step(const Geometry& g, int step);
hipError_t launch_reuse_mask(const Geometry& g, int step, const retro_kv_cache& c,
                             const retro_selection& sel, hipStream_t s);
hipError_t launch_topk_mask(const Geometry& g, int step, const float* scores,
                            const retro_kv_cache& c, const retro_selection& sel,
                            int32_t* sel_phys, hipStream_t s);
hipError_t launch_attend(const Geometry& g, int step, const void* q_window,
                         const retro_kv_cache& c, const retro_selection& sel,
                         const int32_t* sel_phys, float* o_ws, float* l_ws, const void* dummy,
                         hipStream_t s);
// Attention with the page selection (top-k + Alg. 2's mask) computed by each
// of its workgroups (attend_selects(g)); writes the selection outputs (rows,
// mask, physical pages, count) but not last_loaded: the combine launch after
// it takes `selected` = sel.selected and `tok_out` to update it.  scores: the
// score launch's page scores; tok_out: [batch * h_k] ints of workspace.
bool attend_selects(const Geometry& g);
hipError_t launch_attend_select(const Geometry& g, int step, const void* q_window,
                                const retro_kv_cache& c, const retro_selection& sel,
                                int32_t* sel_phys, const float* scores, float* o_ws, float* l_ws,
                                int32_t* tok_out, const void* dummy, hipStream_t s);
// Page scores (+ the token's append), selection, attention and (with o_out)
// the combine + merge of a step in one launch (step_attend.hip): the
// workgroups of a KV head score its pages, publish them as tagged words, each
// reads them all and selects, attends its split, publishes the split's
// log-normalisers as tagged words, and then combines a share of the head's rows
// with the output cache; the head's first workgroup applies the last_loaded
// update, and the sequence's first advances seq_lens (with g.token_pending).
// Only when every workgroup is resident at once (step_attend_supported:
// occupancy times compute units; rtw == 1, max_pages <= 4480, at most 160 pages
// scored per workgroup, at most 64 workgroups per head and 64 KV heads, at most
// kCtlLines workgroups).  Uses the workspace's tagged words and per-workgroup
// control lines (zero-filled once, then holding the last launch's epoch;
// refused with the error word set if last used with another geometry); err: set if a wait ran past spin_limit polls (tag_bias != 0
// makes every wait give up, for tests).  Without o_out, only the partials are
// written (o_ws, l_ws), with the selection, and last_loaded is left as it is.
bool step_attend_supported(const Geometry& g);
int step_attend_workgroups(const Geometry& g);
hipError_t launch_step_attend(const Geometry& g, int step, const void* q_window, const void* k_new,
                              const void* v_new, const retro_kv_cache& c,
                              const retro_selection& sel, void* workspace, float* o_ws,
                              float* l_ws, int32_t* tok_out, int32_t* err, int spin_limit,
                              uint32_t tag_bias, const retro_output_cache* oc, float* o_out,
                              float* lse_out, hipStream_t s);
int compute_units();
// mode 0: combine splits -> o_part/lse_part; 1: o_part -> output cache; 2: splits -> cache
// With g.token_pending and a cache, the launch also advances seq_lens past the
// step's token (when its page is mapped).  With `selected` and `tok_upd` (from
// launch_attend_select; num_selected and cache required), it also applies the
// step's last_loaded update.  With `err` (mode 2), rows are written as NaN if
// that word is set (a bounded wait of the launch before ran out).
hipError_t launch_combine_merge(const Geometry& g, int step, int mode, const float* o_ws,
                                const float* l_ws, const int32_t* num_selected,
                                const float* o_part, const float* l_part, float* o_part_out,
                                float* l_part_out, const retro_output_cache* oc, float* o_out,
                                float* lse_out, const retro_kv_cache* cache, hipStream_t s,
                                const int32_t* selected = nullptr,
                                const int32_t* tok_upd = nullptr,
                                const int32_t* err = nullptr);

}  // namespace retro
