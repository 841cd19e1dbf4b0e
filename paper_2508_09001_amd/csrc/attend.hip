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
  __shared__ int s_tok;
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
      s_page, s_mask, &s_tok, -1, [] {}, SelectionRows{});
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
  __shared__ int s_k, s_tok;
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
      s_mask, &s_tok, -1, select, [&](int t, int, int& lp, int& m, int& phys) {
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
  if (mp <= 6 * kAttendThreads) return attend_select_p<T, D, 6>(a, ta, tok_out, s);
  if (mp <= 9 * kAttendThreads) return attend_select_p<T, D, 9>(a, ta, tok_out, s);
  return attend_select_p<T, D, 12>(a, ta, tok_out, s);
}

}  // namespace

int attend_min_waves(int dtype, int D) {
  const int pieces = dtype == RETRO_BF16 ? (D == 128 ? Tiles<bf16_t, 128>::PIECES : Tiles<bf16_t, 64>::PIECES)
                                         : (D == 128 ? Tiles<float, 128>::PIECES : Tiles<float, 64>::PIECES);
  return (pieces + 64 * kMaxPieces - 1) / (64 * kMaxPieces);
}

AttendArgs make_attend_args(const Geometry& g, int step, const void* q_window,
                            const retro_kv_cache& c, const retro_selection& sel,
                            const int32_t* sel_phys, float* o_ws, float* l_ws, const void* dummy) {
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
  a.dummy = dummy;
  a.tok_k = nullptr;
  a.tok_v = nullptr;
  return a;
}

hipError_t launch_attend(const Geometry& g, int step, const void* q_window,
                         const retro_kv_cache& c, const retro_selection& sel,
                         const int32_t* sel_phys, float* o_ws, float* l_ws, const void* dummy,
                         hipStream_t s) {
  if (!dummy) return hipErrorInvalidValue;
  const AttendArgs a = make_attend_args(g, step, q_window, c, sel, sel_phys, o_ws, l_ws, dummy);
  if (g.dtype == RETRO_BF16) return g.D == 128 ? attend_d<bf16_t, 128>(a, s) : attend_d<bf16_t, 64>(a, s);
  return g.D == 128 ? attend_d<float, 128>(a, s) : attend_d<float, 64>(a, s);
}

bool attend_selects(const Geometry& g) { return g.max_pages <= 12 * kAttendThreads; }

hipError_t launch_attend_select(const Geometry& g, int step, const void* q_window,
                                const retro_kv_cache& c, const retro_selection& sel,
                                int32_t* sel_phys, const float* scores, float* o_ws, float* l_ws,
                                int32_t* tok_out, const void* dummy, hipStream_t s) {
  if (!attend_selects(g) || !sel_phys || !tok_out || !dummy) return hipErrorInvalidValue;
  const AttendArgs a = make_attend_args(g, step, q_window, c, sel, sel_phys, o_ws, l_ws, dummy);
  const TopkArgs ta{g, step, scores, c.page_table, c.last_loaded, sel.selected, sel.mask,
                    sel.num_selected, sel_phys};
  if (g.dtype == RETRO_BF16)
    return g.D == 128 ? attend_select_d<bf16_t, 128>(a, ta, tok_out, s)
                      : attend_select_d<bf16_t, 64>(a, ta, tok_out, s);
  return g.D == 128 ? attend_select_d<float, 128>(a, ta, tok_out, s)
                    : attend_select_d<float, 64>(a, ta, tok_out, s);
}

}  // namespace retro
