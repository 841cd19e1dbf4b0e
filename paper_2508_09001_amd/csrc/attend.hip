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
  attend_role<T, D, RTW, MAXP, RTW == 1, false>(a, b, h, rg, split, [&] { return live_seq_len(g, a.seq_lens, a.pt, b); },
                         lds, s_phys, s_page, s_mask, [] {});
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

}  // namespace retro
