// One attention pass over the selected pages for the W+1 queries of the
// retrospective window (Alg. 1 "Attention"; eq. update-org for the current
// query, eq. update-sup for the past ones, masked as in the "Retrospective Mask"
// paragraph: row tau uses page p iff tau == t or M_p < tau).
//
// Work decomposition.  A workgroup owns one (sequence, KV head, split), a split
// being a run of consecutive entries of the selected-page list, processed as
// 32-token chunks (two 16-token tiles: two pages of 16, or one page of 32).
// Every chunk's keys and values are read from HBM once, staged in LDS, and used
// by all R = (W+1)*G rows of the KV head's group (row = window step r times G
// plus query head), so the gather is shared by the whole window and group.
// Rows are split into 16-row tiles; each wavefront owns RTW row tiles.
//
// Per chunk and row tile, on MFMA (gfx950):
//   S^T (16 tokens x 16 rows) = K (16 x d) . Q^T (d x 16), per 16-token tile
//       bf16: v_mfma_f32_16x16x32_bf16, d/32 steps;  f32: 16x16x4, d/4 steps
//   masking, online softmax in registers (exp2 domain, running max per row)
//   O^T (16 d x 16 rows) += V^T (16 d x 32 tokens) . P^T (32 tokens x 16 rows)
//       bf16: P is split into bf16 hi + lo parts (two MFMAs) so that rounding P
//             to bf16 does not cost accuracy; f32: 16x16x4.
// The S^T accumulator layout (lane l: row l%16, tokens 4*(l/16)..+3) is exactly
// the B operand layout of the PV product once the 32 chunk tokens are ordered
// as [tile 0: 4g..4g+3, tile 1: 4g..4g+3] for lane group g; V^T is read from LDS
// in the same token order, so no data moves between lanes.  The running max is
// per row, i.e. per lane column, and the O^T accumulator keeps the row in the
// lane column too, so rescaling needs no shuffles.
//
// Values live d-major in the cache (v_cache[page][h][d][P]), which is what makes
// the PV operand a contiguous LDS read.
//
// Output: per split and row, the normalised partial output and its natural-log
// normaliser, combined across splits by the merge kernel.
#include <cstdlib>

#include "roles.h"

namespace retro {
namespace {

// Workgroups have eight wavefronts (the host checks); staging registers are
// sized for that: a chunk's 16-byte pieces spread over 512 threads.
constexpr int kAttendThreads = 512;

template <typename T, int D, int RTW>
__global__ void __launch_bounds__(kAttendThreads) attend_kernel(AttendArgs a) {
  using TL = Tiles<T, D>;
  constexpr int MAXP = (TL::PIECES + kAttendThreads - 1) / kAttendThreads;
  __shared__ __attribute__((aligned(16))) T lds[2 * TL::BUF_ELEMS];
  __shared__ int s_phys[kMaxSplitPages];
  __shared__ int s_page[kMaxSplitPages];
  __shared__ int s_mask[kMaxSplitPages];
  const Geometry& g = a.g;
  // Work units are ordered (sequence, KV head, row group, split), split fastest,
  // and spread so that the units of one KV head share an XCD (workgroups go to
  // the 8 XCDs round-robin): its partial outputs then stay in that XCD's L2 for
  // the combine.
  int u = xcd_remap(blockIdx.x, gridDim.x);
  const int split = u % g.n_splits;
  u /= g.n_splits;
  const int rg = u % g.n_rgroups;
  u /= g.n_rgroups;
  const int h = u % g.hk, b = u / g.hk;
  attend_role<T, D, RTW, MAXP, RTW == 1, false>(
      a, b, h, rg, split, [&] { return live_seq_len(g, a.seq_lens, a.pt, b); }, lds, s_phys,
      s_page, s_mask, [] {}, SelectionRows{});
}

template <typename T, int D, int RTW>
hipError_t attend_t(const AttendArgs& a, hipStream_t s) {
  const Geometry& g = a.g;
  const int64_t n = (int64_t)g.n_splits * g.n_rgroups * g.hk * g.batch;
  if (64 * g.waves != kAttendThreads) return hipErrorInvalidValue;
  attend_kernel<T, D, RTW><<<(unsigned)n, kAttendThreads, 0, s>>>(a);
  return hipGetLastError();
}

template <typename T, int D>
hipError_t attend_d(const AttendArgs& a, hipStream_t s) {
  return a.g.rtw == 1 ? attend_t<T, D, 1>(a, s) : attend_t<T, D, 2>(a, s);
}

// The selection of KV head bh as every attention workgroup of the head runs it
// (topk_core over the head's scores, the same result in each): slots [first,
// first + pages_per_split) of the kept pages go to l_lp / l_m / l_ph (logical
// page, mask value, physical page) and the count to *s_k; the `writer`
// workgroup also writes the selection rows (-1 past the count), the count, and
// tok_out[bh] = the step token's page if it is not kept, else -1.  Ends with a
// barrier.  len_of / tok_lp / wait as for topk_core.
template <int PER, typename LenOf, typename Wait>
__device__ __forceinline__ void select_for_split(const TopkArgs& ta, int bh, int first, bool writer,
                                                 LenOf&& len_of, const int& tok_lp,
                                                 Wait&& wait, char* lds,
                                                 int (&l_lp)[kMaxSplitPages],
                                                 int (&l_m)[kMaxSplitPages],
                                                 int (&l_ph)[kMaxSplitPages], int& s_k,
                                                 int32_t* tok_out) {
  const Geometry& g = ta.g;
  const int tid = thread_index();
  uint32_t* hist = reinterpret_cast<uint32_t*>(lds);
  int* small = reinterpret_cast<int*>(hist + kTopkHistWords);
  int32_t* sel_row = ta.selected + (int64_t)bh * g.k_max;
  int32_t* m_row = ta.mask + (int64_t)bh * g.k_max;
  int32_t* ph_row = ta.sel_phys + (int64_t)bh * g.k_max;
  const int k = topk_core<PER, kAttendThreads / 64>(
      ta, bh, len_of, tok_lp, hist, small, wait, [&](int pos, int p, int a_old, int phys) {
        const int ph = (phys >= 0 && phys < g.num_phys) ? phys : -1;
        if (pos >= first && pos < first + g.pages_per_split) {
          l_lp[pos - first] = p;
          l_m[pos - first] = a_old;
          l_ph[pos - first] = ph;
        }
        if (writer) {
          if (pos >= 0) {
            sel_row[pos] = p;
            m_row[pos] = a_old;
            ph_row[pos] = ph;
          }
          if (p == tok_lp) tok_out[bh] = pos < 0 ? p : -1;
        }
      });
  if (writer) {
    for (int i = k + tid; i < g.k_max; i += kAttendThreads) {
      sel_row[i] = -1;
      m_row[i] = -1;
      ph_row[i] = -1;
    }
    if (tid == 0) {
      ta.num_selected[bh] = k;
      if (tok_lp < 0) tok_out[bh] = -1;
    }
  }
  if (tid == 0) s_k = k;
  __syncthreads();  // the split's page list and the count are in LDS
}

// Attention with the page selection in front: every workgroup of a KV head
// runs the head's top-k (the same computation on the same scores, so the same
// result) and takes its split's slots of the selection from LDS, instead of
// waiting for a selection launch and reading the rows back.  The workgroup of
// split 0, row group 0 writes the selection rows, the count and, for the
// step's token page, -1 when it is kept and its logical page otherwise
// (tok_out[bh]); last_loaded is left alone here (other workgroups of the head
// read it) and updated by the combine launch from those outputs.  The
// selection's histograms share LDS with the chunk staging, which is only used
// after the page list is in place.
template <typename T, int D, int RTW, int PER>
__global__ void __launch_bounds__(kAttendThreads) attend_select_kernel(AttendArgs a, TopkArgs ta,
                                                                       int32_t* tok_out) {
  using TL = Tiles<T, D>;
  constexpr int MAXP = (TL::PIECES + kAttendThreads - 1) / kAttendThreads;
  constexpr int kStageBytes = 2 * TL::BUF_ELEMS * (int)sizeof(T);
  constexpr int kSelectBytes = (kTopkHistWords + kTopkSmall) * 4;
  __shared__ __attribute__((aligned(16))) char lds[std::max(kStageBytes, kSelectBytes)];
  __shared__ int s_phys[kMaxSplitPages];
  __shared__ int s_page[kMaxSplitPages];
  __shared__ int s_mask[kMaxSplitPages];
  __shared__ int l_lp[kMaxSplitPages], l_m[kMaxSplitPages], l_ph[kMaxSplitPages];
  __shared__ int s_k;
  const Geometry& g = a.g;
  int u = xcd_remap(blockIdx.x, gridDim.x);
  const int split = u % g.n_splits;
  u /= g.n_splits;
  const int rg = u % g.n_rgroups;
  u /= g.n_rgroups;
  const int h = u % g.hk, b = u / g.hk;
  const int bh = b * g.hk + h;
  const bool writer = split == 0 && rg == 0;
  const int first = split * g.pages_per_split;
  int seq_len = 0, tok_lp = -1;
  auto select = [&] {
    select_for_split<PER>(
        ta, bh, first, writer,
        [&] {
          const int pos = a.seq_lens[b];
          seq_len = pos;
          tok_lp = -1;
          if (g.token_pending && token_phys(g, a.pt, b, pos) >= 0) {
            seq_len = pos + 1;
            tok_lp = pos / g.P;
          }
          return seq_len;
        },
        tok_lp, [] {}, lds, l_lp, l_m, l_ph, s_k, tok_out);
  };
  attend_role<T, D, RTW, MAXP, RTW == 1, false>(
      a, b, h, rg, split, [&] { return seq_len; }, reinterpret_cast<T*>(lds), s_phys, s_page,
      s_mask, select, [&](int t, int, int& lp, int& m, int& phys) {
        if (t < g.pages_per_split) {
          lp = l_lp[t];
          m = l_m[t];
          phys = l_ph[t];
        }
        return s_k;
      });
}

template <typename T, int D, int PER>
hipError_t attend_select_p(const AttendArgs& a, const TopkArgs& ta, int32_t* tok_out,
                           hipStream_t s) {
  const Geometry& g = a.g;
  const int64_t n = (int64_t)g.n_splits * g.n_rgroups * g.hk * g.batch;
  if (64 * g.waves != kAttendThreads || g.max_pages > PER * kAttendThreads) return hipErrorInvalidValue;
  if (g.rtw == 1)
    attend_select_kernel<T, D, 1, PER><<<(unsigned)n, kAttendThreads, 0, s>>>(a, ta, tok_out);
  else
    attend_select_kernel<T, D, 2, PER><<<(unsigned)n, kAttendThreads, 0, s>>>(a, ta, tok_out);
  return hipGetLastError();
}

template <typename T, int D>
hipError_t attend_select_d(const AttendArgs& a, const TopkArgs& ta, int32_t* tok_out,
                           hipStream_t s) {
  const int mp = a.g.max_pages;
  if (mp <= 2 * kAttendThreads) return attend_select_p<T, D, 2>(a, ta, tok_out, s);
  if (mp <= 5 * kAttendThreads) return attend_select_p<T, D, 5>(a, ta, tok_out, s);
  return attend_select_p<T, D, 12>(a, ta, tok_out, s);
}

// Scoring in the same launch (see attend_full_kernel).
struct ScoreInArgs {
  const void* q;      // current query rows: sequence b's at q + b * q_bstride
  int64_t q_bstride;  // elements
  void* dg;           // digests
  float* scores;      // [batch][h_k][max_pages]
  const void* k_new;  // the step's token, [batch][h_k][d]
  const void* v_new;
  uint64_t* cnt;      // per KV head: an arrival counter, a 128-byte line each
  int32_t* err;       // set when a wait runs past its bound
  int ppb;            // pages scored per workgroup
  int spin_limit;     // polls before a wait gives up
  uint64_t target_bias;  // added to every wait's target (a test makes waits time out with it)
};

// Page scores, the token's append, the selection and the attention in one
// launch.  Each workgroup of a KV head scores its share of the head's pages
// (appending the token if its page is in that share), writes the scores (and
// the token) device-coherently, waits for its own stores, meets at a barrier
// and counts itself in on the head's arrival counter; then it polls the counter
// until the whole head has arrived, and runs the selection and attention as
// attend_select_kernel does.  The host launches this form only when every
// workgroup fits on the chip at once (no more workgroups than compute units,
// one per unit), so every wait ends; it is bounded all the same (past
// kSpinLimit polls the error word is set and the workgroup goes on).
// The counter is never reset: it grows by the head's workgroup count every
// launch (64 bits).  Every arrival of a launch precedes every arrival of the
// next one, which starts after it ends, so a count read by a workgroup of the
// launch before it counts itself in lies in [n * c, n * c + c - 1] (c: the
// head's workgroups, n: the launches before) and the workgroup waits for the
// next multiple of c.  Reading it at the start takes the round trip of a
// returning atomic off the path of the head's last arrival; resetting the
// counter instead would take a second counter whose returning atomic kept the
// selection's first wavefront waiting about a microsecond.
template <typename T, int D, int PER, int SITERS, int GC>
__global__ void __launch_bounds__(kAttendThreads) attend_full_kernel(AttendArgs a, TopkArgs ta,
                                                                     ScoreInArgs sc,
                                                                     int32_t* tok_out) {
  using TL = Tiles<T, D>;
  constexpr int MAXP = (TL::PIECES + kAttendThreads - 1) / kAttendThreads;
  constexpr int kStageBytes = 2 * TL::BUF_ELEMS * (int)sizeof(T);
  constexpr int kSelectBytes = (kTopkHistWords + kTopkSmall) * 4;
  __shared__ __attribute__((aligned(16))) char lds[std::max(kStageBytes, kSelectBytes)];
  __shared__ int s_phys[kMaxSplitPages];
  __shared__ int s_page[kMaxSplitPages];
  __shared__ int s_mask[kMaxSplitPages];
  __shared__ int l_lp[kMaxSplitPages], l_m[kMaxSplitPages], l_ph[kMaxSplitPages];
  __shared__ int s_k;
  const Geometry& g = a.g;
  int u = xcd_remap(blockIdx.x, gridDim.x);
  const int split = u % g.n_splits;
  u /= g.n_splits;
  const int rg = u % g.n_rgroups;
  u /= g.n_rgroups;
  const int h = u % g.hk, b = u / g.hk;
  const int bh = b * g.hk + h;
  const int per_head = g.n_splits * g.n_rgroups;
  const bool writer = split == 0 && rg == 0;
  const int first = split * g.pages_per_split;
  const int tid = thread_index();
  uint64_t* arrive = sc.cnt + (int64_t)bh * (kSelCounterInts / 2);
  // thread 0: the head's arrival count before this workgroup counts itself in,
  // read now so that counting in needs no returning atomic (see below)
  uint64_t before = 0, target = 0;
  if (tid == 0) before = __hip_atomic_load(arrive, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);

  // ---- this workgroup's share of the head's page scores
  int seq_len = 0, tok_lp = -1, n_pages = 0;
  {
    const int page0 = (rg * g.n_splits + split) * sc.ppb;
    const int page_end = min(page0 + sc.ppb, g.max_pages);
    score_role<T, D, SITERS, true, GC>(
        g, page0, page_end,
        reinterpret_cast<const T*>(sc.q) + b * sc.q_bstride + (int64_t)h * g.G * D,
        reinterpret_cast<T*>(sc.dg) + (int64_t)bh * g.max_pages * 2 * D,
        sc.scores + (int64_t)bh * g.max_pages, reinterpret_cast<float*>(lds),
        [&](int& np) {
          const int pos = a.seq_lens[b];
          StepToken<T> tk{-1, 0, nullptr, nullptr, nullptr, nullptr};
          seq_len = pos;
          if (g.token_pending) {
            const int phys = token_phys(g, a.pt, b, pos);
            if (phys >= 0) {
              seq_len = pos + 1;
              tk = make_step_token<T>(g, b, h, pos, phys, sc.k_new, sc.v_new,
                                      const_cast<void*>(a.kc), const_cast<void*>(a.vc));
            }
          }
          np = n_pages = min((seq_len + g.P - 1) / g.P, g.max_pages);
          tok_lp = tk.lp;
          return tk;
        });
    __builtin_amdgcn_s_waitcnt(0);  // this wavefront's score and token stores have completed
    __syncthreads();
    if (tid == 0) {
      __hip_atomic_fetch_add(arrive, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      target = (before / per_head + 1) * per_head + sc.target_bias;
    }
  }

  // the head's arrival wait, run by the selection once its last_loaded and
  // page-table loads are in flight and its histograms are cleared
  auto head_wait = [&] {
    if (tid == 0) {
      int it = 0;
      while (__hip_atomic_load(arrive, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
        if (++it > sc.spin_limit) {
          __hip_atomic_store(sc.err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          break;
        }
        __builtin_amdgcn_s_sleep(8);  // ~0.2 us between polls
      }
    }
    __syncthreads();
  };
  auto select = [&] {
    select_for_split<PER>(ta, bh, first, writer, [&] { return seq_len; }, tok_lp, head_wait,
                          lds, l_lp, l_m, l_ph, s_k, tok_out);
  };
  attend_role<T, D, 1, MAXP, true, false>(
      a, b, h, rg, split, [&] { return seq_len; }, reinterpret_cast<T*>(lds), s_phys, s_page,
      s_mask, select, [&](int t, int, int& lp, int& m, int& phys) {
        if (t < g.pages_per_split) {
          lp = l_lp[t];
          m = l_m[t];
          phys = l_ph[t];
        }
        return s_k;
      });
}

template <typename T, int D, int PER>
hipError_t attend_full_p(const AttendArgs& a, const TopkArgs& ta, const ScoreInArgs& sc,
                         int32_t* tok_out, hipStream_t s) {
  const Geometry& g = a.g;
  const int64_t n = (int64_t)g.n_splits * g.n_rgroups * g.hk * g.batch;
  if (64 * g.waves != kAttendThreads || g.rtw != 1 || g.max_pages > PER * kAttendThreads ||
      sc.ppb < 1 || sc.ppb > 3 * (kAttendThreads / 64) * 4)
    return hipErrorInvalidValue;
  // the headline group size (4 query heads per KV head) gets an unrolled score loop
  if (g.G == 4)
    attend_full_kernel<T, D, PER, 3, 4><<<(unsigned)n, kAttendThreads, 0, s>>>(a, ta, sc, tok_out);
  else
    attend_full_kernel<T, D, PER, 3, 0><<<(unsigned)n, kAttendThreads, 0, s>>>(a, ta, sc, tok_out);
  return hipGetLastError();
}

template <typename T, int D>
hipError_t attend_full_d(const AttendArgs& a, const TopkArgs& ta, const ScoreInArgs& sc,
                         int32_t* tok_out, hipStream_t s) {
  if (a.g.max_pages <= 2 * kAttendThreads) return attend_full_p<T, D, 2>(a, ta, sc, tok_out, s);
  return attend_full_p<T, D, 5>(a, ta, sc, tok_out, s);
}

}  // namespace

int attend_min_waves(int dtype, int D) {
  const int pieces = dtype == RETRO_BF16 ? (D == 128 ? Tiles<bf16_t, 128>::PIECES : Tiles<bf16_t, 64>::PIECES)
                                         : (D == 128 ? Tiles<float, 128>::PIECES : Tiles<float, 64>::PIECES);
  return (pieces + 64 * kMaxPieces - 1) / (64 * kMaxPieces);
}

AttendArgs make_attend_args(const Geometry& g, int step, const void* q_window,
                            const retro_kv_cache& c, const retro_selection& sel,
                            const int32_t* sel_phys, float* o_ws, float* l_ws) {
  AttendArgs a;
  a.g = g;
  a.step = step;
  a.scale_log2 = g.sm_scale * kLog2e;
  a.q = q_window;
  a.kc = c.k_cache;
  a.vc = c.v_cache;
  a.pt = c.page_table;
  a.seq_lens = c.seq_lens;
  a.sel = sel.selected;
  a.msk = sel.mask;
  a.nsel = sel.num_selected;
  a.sel_phys = sel_phys;
  a.o_ws = o_ws;
  a.l_ws = l_ws;
  return a;
}

hipError_t launch_attend(const Geometry& g, int step, const void* q_window,
                         const retro_kv_cache& c, const retro_selection& sel,
                         const int32_t* sel_phys, float* o_ws, float* l_ws, hipStream_t s) {
  const AttendArgs a = make_attend_args(g, step, q_window, c, sel, sel_phys, o_ws, l_ws);
  if (g.dtype == RETRO_BF16) return g.D == 128 ? attend_d<bf16_t, 128>(a, s) : attend_d<bf16_t, 64>(a, s);
  return g.D == 128 ? attend_d<float, 128>(a, s) : attend_d<float, 64>(a, s);
}

bool attend_selects(const Geometry& g) { return g.max_pages <= 12 * kAttendThreads; }

hipError_t launch_attend_select(const Geometry& g, int step, const void* q_window,
                                const retro_kv_cache& c, const retro_selection& sel,
                                int32_t* sel_phys, const float* scores, float* o_ws, float* l_ws,
                                int32_t* tok_out, hipStream_t s) {
  if (!attend_selects(g) || !sel_phys || !tok_out) return hipErrorInvalidValue;
  const AttendArgs a = make_attend_args(g, step, q_window, c, sel, sel_phys, o_ws, l_ws);
  const TopkArgs ta{g, step, scores, c.page_table, c.last_loaded, sel.selected, sel.mask,
                    sel.num_selected, sel_phys};
  if (g.dtype == RETRO_BF16)
    return g.D == 128 ? attend_select_d<bf16_t, 128>(a, ta, tok_out, s)
                      : attend_select_d<bf16_t, 64>(a, ta, tok_out, s);
  return g.D == 128 ? attend_select_d<float, 128>(a, ta, tok_out, s)
                    : attend_select_d<float, 64>(a, ta, tok_out, s);
}

bool attend_full_supported(const Geometry& g, int compute_units) {
  const int per_head = g.n_splits * g.n_rgroups;
  const int ppb = (g.max_pages + per_head - 1) / per_head;
  // the score role loads the group's queries as at most two 16-byte pieces per
  // thread and keeps them in LDS as fp32 (within the selection's share)
  const bool q_fits = g.G * g.D <= 2 * kAttendThreads * (16 / g.elt) &&
                      g.G * g.D <= kTopkHistWords + kTopkSmall;
  return q_fits && g.rtw == 1 && g.max_pages <= 5 * kAttendThreads &&
         ppb <= 3 * (kAttendThreads / 64) * 4 && (int64_t)per_head * g.hk * g.batch <= compute_units;
}

hipError_t launch_attend_full(const Geometry& g, int step, const void* q_window, const void* k_new,
                              const void* v_new, const retro_kv_cache& c,
                              const retro_selection& sel, int32_t* sel_phys, float* scores,
                              float* o_ws, float* l_ws, int32_t* tok_out, uint64_t* counters,
                              int32_t* err, hipStream_t s) {
  if (!sel_phys || !tok_out || !counters || !err) return hipErrorInvalidValue;
  const AttendArgs a = make_attend_args(g, step, q_window, c, sel, sel_phys, o_ws, l_ws);
  const TopkArgs ta{g, step, scores, c.page_table, c.last_loaded, sel.selected, sel.mask,
                    sel.num_selected, sel_phys};
  ScoreInArgs sc;
  sc.q = (const char*)q_window + (int64_t)g.W * g.hq * g.D * g.elt;
  sc.q_bstride = (int64_t)(g.W + 1) * g.hq * g.D;
  sc.dg = c.digest;
  sc.scores = scores;
  sc.k_new = k_new;
  sc.v_new = v_new;
  sc.cnt = counters;
  sc.err = err;
  const int per_head = g.n_splits * g.n_rgroups;
  sc.ppb = (g.max_pages + per_head - 1) / per_head;
  // RETRO_TEST_WAIT_TIMEOUT=1 (tests of the failure path): every wait gives up
  // after a few polls, its target being out of reach
  const char* t = std::getenv("RETRO_TEST_WAIT_TIMEOUT");
  const bool timeout = t && t[0] == '1';
  sc.spin_limit = timeout ? 4 : kSpinLimit;
  sc.target_bias = timeout ? (1ull << 40) : 0ull;
  if (g.dtype == RETRO_BF16)
    return g.D == 128 ? attend_full_d<bf16_t, 128>(a, ta, sc, tok_out, s)
                      : attend_full_d<bf16_t, 64>(a, ta, sc, tok_out, s);
  return g.D == 128 ? attend_full_d<float, 128>(a, ta, sc, tok_out, s)
                    : attend_full_d<float, 64>(a, ta, sc, tok_out, s);
}

}  // namespace retro
