// The whole decode step in one launch: AppendKV + page scores, top-k + mask,
// attention, combine + merge (Alg. 1 without its UpdateKV step).
//
// Each KV head of the batch (bh = b * h_k + h) belongs to lane bh mod 8.  A lane
// has its own ticket counter; the workgroups with blockIdx mod 8 == lane (those
// the dispatcher sends to one XCD) take tickets from it in the order they start,
// and ticket order is task order:
//   [score blocks of the lane's heads] [top-k of each head] [attention splits]
//   [combine + merge blocks]
// A task waits only for earlier tasks of its own head, i.e. for workgroups that
// took smaller tickets of the same lane and therefore have started: the
// schedule cannot deadlock whatever the number of resident workgroups, and all
// of one head's traffic (scores, selection, partial outputs) stays in one XCD's
// L2.  Hand-offs use per-head counters (roles.h: block_signal / block_wait,
// bounded waits).
//
// Workgroups have kFusedWaves (8) wavefronts and at most 128 VGPRs per lane, so
// two fit on a CU: at the workloads' sizes every task of an XCD is resident
// from the start, and consumers issue the loads that do not depend on their
// producer (queries, page table, last_loaded) before they wait.
//
// The step's own token is appended by the score block whose pages include it,
// before that block scores them.  Sequence lengths are advanced by the last
// workgroup to finish, which also zeroes every synchronisation word, so the
// workspace is ready for the next launch.
#include "roles.h"

namespace retro {

AttendArgs make_attend_args(const Geometry& g, int step, const void* q_window,
                            const retro_kv_cache& c, const retro_selection& sel,
                            const int32_t* sel_phys, float* o_ws, float* l_ws);
MergeArgs make_merge_args(const Geometry& g, int step, int mode, const float* o_ws,
                          const float* l_ws, const int32_t* num_selected, const float* o_part,
                          const float* l_part, float* o_part_out, float* l_part_out,
                          const retro_output_cache* oc, float* o_out, float* lse_out);

namespace {

constexpr int kMaxLanes = 8;  // lanes: workgroups with blockIdx mod 8 == lane share an XCD
constexpr int kTopkPer = 12;

struct StepArgs {
  Geometry g;
  int step;
  AttendArgs at;
  TopkArgs tk;
  MergeArgs mg;
  const void* q_cur;  // row W of the query window
  int64_t q_bstride;
  const void* k_new;
  const void* v_new;
  void* kc;
  void* vc;
  void* dg;
  const int32_t* pt;
  int32_t* seq_lens;
  int32_t* A;
  float* scores;
  int32_t* ctl;
};

template <typename T, int D>
struct FusedLds {
  static constexpr size_t SCORE = sizeof(float) * 16 * D;
  static constexpr size_t TOPK = sizeof(uint32_t) * kTopkHistWords;
  static constexpr size_t ATTEND = sizeof(T) * 2 * Tiles<T, D>::BUF_ELEMS;
  static constexpr size_t BYTES = ATTEND > TOPK ? (ATTEND > SCORE ? ATTEND : SCORE)
                                                : (TOPK > SCORE ? TOPK : SCORE);
};

constexpr int kThreads = 64 * kFusedWaves;

// PER: stripes of the head's pages per thread in the top-k role (max_pages <= PER * kThreads)
template <typename T, int D, int PER>
__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4, 8)))
step_kernel(StepArgs a) {
  // chunk pieces per thread of the attention role
  constexpr int MAXP = (Tiles<T, D>::PIECES + kThreads - 1) / kThreads;
  __shared__ __attribute__((aligned(16))) char lds[FusedLds<T, D>::BYTES];
  __shared__ int s_phys[kMaxSplitPages];
  __shared__ int s_page[kMaxSplitPages];
  __shared__ int s_mask[kMaxSplitPages];
  __shared__ int small[kTopkSmall];
  __shared__ int s_ticket, s_last;

  const Geometry& g = a.g;
  const int tid = threadIdx.x;
  const int BH = g.batch * g.hk;
  // per-head counters, kCtlStride ints apart: cntX + kCtlStride * bh
  int32_t* cntA = a.ctl + kCtlCounts;
  int32_t* cntB = cntA + BH * kCtlStride;
  int32_t* cntC = cntB + BH * kCtlStride;
  int32_t* err = a.ctl + kCtlError;

  const int lane = blockIdx.x % kMaxLanes;
  if (tid == 0)
    s_ticket = __hip_atomic_fetch_add(a.ctl + kCtlTicket + kCtlStride * lane, 1,
                                      __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  {
    int t = s_ticket;
    const int nbh = (BH - lane + kMaxLanes - 1) / kMaxLanes;  // heads in this lane
    int role = -1, i = 0, sub = 0;
    if (t < nbh * g.fA) {
      role = 0, i = t / g.fA, sub = t % g.fA;
    } else if ((t -= nbh * g.fA) < nbh) {
      role = 1, i = t;
    } else if ((t -= nbh) < nbh * g.fC) {
      role = 2, i = t / g.fC, sub = t % g.fC;
    } else if ((t -= nbh * g.fC) < nbh * g.fD) {
      role = 3, i = t / g.fD, sub = t % g.fD;
    }

    if (role >= 0) {
      const int bh = lane + kMaxLanes * i;
      const int b = bh / g.hk, h = bh - b * g.hk;
      // the step's token goes to position seq_lens[b] if its logical page is mapped
      const int pos = a.seq_lens[b];
      const int lp = pos / g.P;
      const int phys_tok = token_phys(g, a.pt, b, pos);
      const bool tok_ok = phys_tok >= 0;
      const int seq_len = pos + (tok_ok ? 1 : 0);
      const int n_pages = min((seq_len + g.P - 1) / g.P, g.max_pages);

      if (role == 0) {
        StepToken<T> tk{-1, 0, nullptr, nullptr, nullptr, nullptr};
        if (tok_ok)
          tk = make_step_token<T>(g, b, h, pos, phys_tok, a.k_new, a.v_new, a.kc, a.vc);
        const int ppb = kFusedWaves * ScoreShape<T, D>::PPW * kFusedScoreIters;
        score_role<T, D, kFusedScoreIters, true>(
            g, sub * ppb, min(sub * ppb + ppb, g.max_pages),
            reinterpret_cast<const T*>(a.q_cur) + b * a.q_bstride + (int64_t)h * g.G * D,
            reinterpret_cast<T*>(a.dg) + (int64_t)bh * g.max_pages * 2 * D,
            a.scores + (int64_t)bh * g.max_pages, reinterpret_cast<float*>(lds),
            [&](int& np) { np = n_pages; return tk; });
        block_signal(cntA + kCtlStride * bh);
      } else if (role == 1) {
        topk_role<PER, kFusedWaves, true>(a.tk, bh, [&] { return seq_len; }, tok_ok ? lp : -1,
                                  reinterpret_cast<uint32_t*>(lds), small,
                                  [&] { block_wait(cntA + kCtlStride * bh, g.fA, err); });
        block_signal(cntB + kCtlStride * bh);
      } else if (role == 2) {
        const int rg = sub / g.n_splits, split = sub - rg * g.n_splits;
        attend_role<T, D, 1, MAXP, false, true>(a.at, b, h, rg, split, [&] { return seq_len; }, reinterpret_cast<T*>(lds), s_phys,
                               s_page, s_mask, [&] { block_wait(cntB + kCtlStride * bh, 1, err); },
                               SelectionRows{});
        block_signal(cntC + kCtlStride * bh);
      } else {
        block_wait(cntC + kCtlStride * bh, g.fC, err);
        const int per_bh = g.G * a.mg.xs;
        const int local = sub * (blockDim.x >> 6) + (tid >> 6);
        if (local < per_bh) merge_unit<D, 8, true>(a.mg, bh * per_bh + local);
      }
    }
  }

  // exit: the last workgroup advances the sequence lengths (no other
  // workgroup reads them any more) and clears the synchronisation words for
  // the next launch (every other workgroup is past its waits)
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (tid == 0) {
    const int old = __hip_atomic_fetch_add(a.ctl + kCtlExit, 1, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT);
    s_last = (old == (int)gridDim.x - 1);
  }
  __syncthreads();
  if (s_last) {
    for (int b = tid; b < g.batch; b += blockDim.x) {
      const int pos = a.seq_lens[b];
      if (token_phys(g, a.pt, b, pos) >= 0) a.seq_lens[b] = pos + 1;
    }
    for (int l = tid; l < kMaxLanes; l += blockDim.x) put_c<true>(a.ctl + kCtlTicket + kCtlStride * l, 0);
    for (int e = tid; e < 3 * BH; e += blockDim.x) put_c<true>(a.ctl + kCtlCounts + kCtlStride * e, 0);
    if (tid == 0) put_c<true>(a.ctl + kCtlExit, 0);
  }
}

template <typename T, int D>
hipError_t step_t(const StepArgs& a, hipStream_t s) {
  if (a.g.max_pages <= kThreads * 6)
    step_kernel<T, D, 6><<<(unsigned)a.g.f_grid, kThreads, 0, s>>>(a);
  else
    step_kernel<T, D, kTopkPer><<<(unsigned)a.g.f_grid, kThreads, 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace

int fused_score_pages_per_block(int dtype, int D) {
  const int ppw = dtype == RETRO_BF16 ? (D == 128 ? ScoreShape<bf16_t, 128>::PPW : ScoreShape<bf16_t, 64>::PPW)
                                      : (D == 128 ? ScoreShape<float, 128>::PPW : ScoreShape<float, 64>::PPW);
  return kFusedWaves * ppw * kFusedScoreIters;
}

bool fused_supported(const Geometry& g) {
  // partial outputs are addressed with 32-bit byte offsets (device-coherent
  // buffer accesses)
  const double part_bytes = (double)g.batch * g.hk * g.n_splits * g.R * g.D * sizeof(float);
  return g.max_pages <= kTopkPer * kThreads && g.G <= 16 && part_bytes < 2147483648.0;
}

hipError_t launch_step_fused(const Geometry& g, int step, const void* q_window, const void* k_new,
                             const void* v_new, const retro_kv_cache& c,
                             const retro_selection& sel, const retro_output_cache* oc,
                             float* o_out, float* lse_out, void* workspace, hipStream_t s) {
  float* scores = reinterpret_cast<float*>((char*)workspace + g.ws_scores);
  int32_t* phys = reinterpret_cast<int32_t*>((char*)workspace + g.ws_phys);
  float* o_ws = reinterpret_cast<float*>((char*)workspace + g.ws_opart);
  float* l_ws = reinterpret_cast<float*>((char*)workspace + g.ws_lpart);
  StepArgs a;
  a.g = g;
  a.step = step;
  // the attention tasks: one row tile per wavefront
  Geometry ga = g;
  ga.rtw = 1;
  ga.waves = kFusedWaves;
  ga.n_rgroups = g.f_rgroups;
  ga.tiles_per_group = g.f_tpg;
  a.at = make_attend_args(ga, step, q_window, c, sel, phys, o_ws, l_ws);
  a.tk = TopkArgs{g, step, scores, c.page_table, c.last_loaded, sel.selected, sel.mask,
                  sel.num_selected, phys};
  a.mg = make_merge_args(g, step, 2, o_ws, l_ws, sel.num_selected, nullptr, nullptr, nullptr,
                         nullptr, oc, o_out, lse_out);
  a.q_cur = (const char*)q_window + (int64_t)g.W * g.hq * g.D * g.elt;
  a.q_bstride = (int64_t)(g.W + 1) * g.hq * g.D;
  a.k_new = k_new;
  a.v_new = v_new;
  a.kc = c.k_cache;
  a.vc = c.v_cache;
  a.dg = c.digest;
  a.pt = c.page_table;
  a.seq_lens = c.seq_lens;
  a.A = c.last_loaded;
  a.scores = scores;
  a.ctl = reinterpret_cast<int32_t*>((char*)workspace + g.ws_ctl);
  if (g.dtype == RETRO_BF16) return g.D == 128 ? step_t<bf16_t, 128>(a, s) : step_t<bf16_t, 64>(a, s);
  return g.D == 128 ? step_t<float, 128>(a, s) : step_t<float, 64>(a, s);
}

}  // namespace retro
