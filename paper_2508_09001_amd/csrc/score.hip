// Page criticality score, eq. (quest_score), per (sequence, KV head, page), in
// the fixed fp32 order described in roles.h (score_role).  Digests are stored
// per logical page, so a KV head's digests form one contiguous stream; a
// workgroup scores a block of consecutive pages, four per wavefront.
//
// With a selection epilogue (PER > 0) the kernel also runs PageSelect and
// UpdateAndBuildMask: the last workgroup of each KV head runs the top-k + mask
// role on the head's scores (see topk.hip for the algorithm), then clears the
// head's counter for the next launch.  That role runs in one workgroup per
// head, so its time is the instruction count of one wavefront: workgroups of
// sixteen wavefronts give each thread at most PER = 1..6 pages of the head.  Scores are written and read with
// device-coherent (agent-scope) atomic stores and loads, which bypass the
// per-XCD L2s; a workgroup counts itself out only after its score stores have
// completed, so the last one reads them all without any L2 write-back or
// invalidation (fences at device scope would write back and invalidate whole
// L2s, once per workgroup).
#include <algorithm>

#include "roles.h"

namespace retro {
namespace {

// Workgroup shape.  Four pages per wavefront and pass, sixteen wavefronts (with
// the selection epilogue, the selection's per-thread share of the head's pages
// is then small), up to two passes: a KV head's pages are spread over as many
// workgroups as fit on the chip at once (one sixteen-wavefront workgroup per
// compute unit), since a workgroup that waits for a free unit starts about
// 1.3 us after one ends (and would hold up its head's selection); a wavefront
// with no page in the second pass skips it.  Without the epilogue (PER == 0:
// the selection runs in the attention launch), eight wavefronts of up to four
// passes (the same 128 pages, more loads in flight per wavefront, two more
// workgroups per compute unit): 70.2 against 71.5 us per layer-step at batch
// 16, 144.9 against 146.6 at the batch-4 long-generation workload.
constexpr int score_threads(int per) { return per == 0 ? 512 : 1024; }
constexpr int score_iters(int per) { return per == 0 ? 4 : 2; }
// most pages a workgroup scores
constexpr int score_pages_per_block(int per) { return score_threads(per) / 64 * 4 * score_iters(per); }


// Workgroups per KV head and pages per workgroup of a score launch.
void select_split(const Geometry& g, int* nbh, int* ppb) {
  const int one_pass = score_threads(1) / 64 * 4;
  const int fit = std::max(1, compute_units() / std::max(1, g.hk * g.batch));
  int n = (g.max_pages + one_pass - 1) / one_pass;
  if (n > fit) n = std::max(fit, (g.max_pages + score_pages_per_block(1) - 1) / score_pages_per_block(1));
  const int per = (g.max_pages + n - 1) / n;
  *ppb = per;
  *nbh = (g.max_pages + per - 1) / per;
}

struct TokenArgs {
  const void* k_new;
  const void* v_new;
  void* kc;
  void* vc;
  const int32_t* pt;
};

struct SelectArgs {
  TopkArgs tk;
  // per KV head: a head counter, then one counter per group of `group`
  // workgroups, each in a 128-byte line of its own (kSelCounterInts apart);
  // zero between launches
  int32_t* count;
  int group;
  int nbh, ppb;  // workgroups per KV head, pages per workgroup (at most score_pages_per_block)
};

template <typename T, int D, int PER>
__global__ void __launch_bounds__(score_threads(PER)) score_kernel(Geometry g, const T* __restrict__ q,
                                                   int64_t q_bstride, T* __restrict__ dg,
                                                   const int32_t* __restrict__ seq_lens,
                                                   float* __restrict__ scores, TokenArgs ta,
                                                   SelectArgs sa, int ppb) {
  // [G][D] fp32 queries while scoring; the top-k histograms and scratch after
  extern __shared__ __attribute__((aligned(16))) float dyn_lds[];
  static_assert(ScoreShape<T, D>::PPW == 4, "four pages per wavefront and pass");
  const int page0 = blockIdx.x * ppb, page_end = min(page0 + ppb, g.max_pages);
  const int b = blockIdx.z, h = blockIdx.y;
  const int64_t bh = (int64_t)b * g.hk + h;
  if constexpr (PER == 0) {
    // a workgroup whose pages all lie past the sequence (the step's token
    // included) has nothing to score: with sequences of mixed lengths the grid,
    // sized for the longest, would otherwise load their stale digests
    if (page0 * g.P > sload(seq_lens + b)) return;  // uniform
  }
  // the step's token and the sequence's pages (after the digest loads are issued)
  int n_pages = 0, tok_lp = -1, live_len = 0;
  auto tok_of = [&](int& np) {
    const int pos = seq_lens[b];
    StepToken<T> tk{-1, 0, nullptr, nullptr, nullptr, nullptr};
    int seq_len = pos;
    if (g.token_pending) {
      const int phys = token_phys(g, ta.pt, b, pos);
      if (phys >= 0) {
        seq_len = pos + 1;
        tk = make_step_token<T>(g, b, h, pos, phys, ta.k_new, ta.v_new, ta.kc, ta.vc);
      }
    }
    np = n_pages = min((seq_len + g.P - 1) / g.P, g.max_pages);
    tok_lp = tk.lp;
    live_len = seq_len;
    return tk;
  };
  int32_t warm_a = 0, warm_p = 0;
  if constexpr (PER > 0) {
    // Fetch this workgroup's last_loaded and page-table entries along with its
    // digests, so that the selection finds them in the caches.
    const int p = page0 + (int)threadIdx.x;
    if (p < page_end) {
      warm_a = sa.tk.A[bh * g.max_pages + p];
      warm_p = sa.tk.pt[(int64_t)b * g.max_pages + p];
    }
  }
  float* srow = scores + bh * g.max_pages;
  score_role<T, D, score_iters(PER), false>(
      g, page0, page_end, q + b * q_bstride + (int64_t)h * g.G * D, dg + bh * g.max_pages * 2 * D,
      dyn_lds, tok_of, [] {},
      // device-coherent store: a later reader of the same launch (the selection)
      // may run on another XCD
      [&](int page, float v) {
        __hip_atomic_store(srow + page, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      });
  if constexpr (PER > 0) {
    asm volatile("" : : "v"(warm_a), "v"(warm_p));  // keeps the two loads
    __shared__ int s_last;
    __builtin_amdgcn_s_waitcnt(0);  // this wavefront's score stores have completed
    __syncthreads();
    // Count out in two levels (a group of workgroups, then the head), so that
    // no counter takes more than max(group, number of groups) updates; with a
    // single group its counter is the head's.
    if (threadIdx.x == 0) {
      const int ngroups = (gridDim.x + sa.group - 1) / sa.group;
      int32_t* head = sa.count + bh * (int64_t)kSelCounterInts * (1 + kSelMaxGroups);
      const int grp = blockIdx.x / sa.group;
      const int in_grp = min(sa.group, (int)gridDim.x - grp * sa.group);
      int32_t* gc = head + kSelCounterInts * (1 + grp);
      bool last = false;
      if (__hip_atomic_fetch_add(gc, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == in_grp - 1) {
        __hip_atomic_store(gc, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        last = ngroups == 1 ||
               __hip_atomic_fetch_add(head, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                   ngroups - 1;
        if (last && ngroups > 1) __hip_atomic_store(head, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      s_last = last;
    }
    __syncthreads();
    if (s_last) {
      uint32_t* hist = reinterpret_cast<uint32_t*>(dyn_lds);
      int* small = reinterpret_cast<int*>(hist + kTopkHistWords);
      topk_role<PER, score_threads(PER) / 64, false>(sa.tk, (int)bh, [&] { return live_len; }, tok_lp, hist, small, [] {});
    }
  }
}

template <typename T, int D, int PER>
hipError_t score_t(const Geometry& g, int step, const void* q, int64_t qbs,
                   const retro_kv_cache& c, const void* k_new, const void* v_new, float* scores,
                   const SelectArgs& sa, hipStream_t s) {
  if (sa.ppb < 1 || sa.ppb > score_pages_per_block(PER) || sa.nbh < 1) return hipErrorInvalidValue;
  dim3 grid(sa.nbh, g.hk, g.batch);
  size_t lds = sizeof(float) * 2 * g.G * D;  // the queries' q+ and q- halves
  if (PER > 0) lds = std::max(lds, sizeof(int32_t) * (kTopkHistWords + kTopkSmall));
  const TokenArgs ta{k_new, v_new, c.k_cache, c.v_cache, c.page_table};
  score_kernel<T, D, PER><<<grid, score_threads(PER), lds, s>>>(g, (const T*)q, qbs, (T*)c.digest, c.seq_lens,
                                                 scores, ta, sa, sa.ppb);
  return hipGetLastError();
}

template <typename T, int D>
hipError_t score_d(const Geometry& g, int step, const void* q, int64_t qbs,
                   const retro_kv_cache& c, const void* k_new, const void* v_new, float* scores,
                   const SelectArgs& sa, hipStream_t s) {
  if (!sa.count) return score_t<T, D, 0>(g, step, q, qbs, c, k_new, v_new, scores, sa, s);
  constexpr int TH = score_threads(1);
  if (g.max_pages <= TH * 1) return score_t<T, D, 1>(g, step, q, qbs, c, k_new, v_new, scores, sa, s);
  if (g.max_pages <= TH * 2) return score_t<T, D, 2>(g, step, q, qbs, c, k_new, v_new, scores, sa, s);
  if (g.max_pages <= TH * 3) return score_t<T, D, 3>(g, step, q, qbs, c, k_new, v_new, scores, sa, s);
  return score_t<T, D, 6>(g, step, q, qbs, c, k_new, v_new, scores, sa, s);
}

}  // namespace

int compute_units() {
  static int cus[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cus[dev] <= 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    cus[dev] = n;
  }
  return cus[dev];
}

bool score_selects(const Geometry& g) { return g.max_pages <= score_threads(1) * 6; }

hipError_t launch_score(const Geometry& g, int step, const void* q_cur, int64_t q_batch_stride,
                        const retro_kv_cache& c, const void* k_new, const void* v_new,
                        float* scores, const retro_selection* sel, int32_t* sel_phys,
                        int32_t* counters, hipStream_t s) {
  SelectArgs sa{};
  if (sel && counters && score_selects(g)) {
    sa.tk = TopkArgs{g, step, scores, c.page_table, c.last_loaded, sel->selected, sel->mask,
                     sel->num_selected, sel_phys};
    sa.count = counters;
    select_split(g, &sa.nbh, &sa.ppb);
    // one counter per head up to 32 workgroups, else groups of at least 16
    sa.group = sa.nbh <= 32 ? sa.nbh : std::max(16, (sa.nbh + kSelMaxGroups - 1) / kSelMaxGroups);
  } else {  // the shape without the selection epilogue: no co-residency to aim for
    const int ppb_max = score_pages_per_block(0);
    const int n = (g.max_pages + ppb_max - 1) / ppb_max;
    sa.ppb = (g.max_pages + n - 1) / n;
    sa.nbh = (g.max_pages + sa.ppb - 1) / sa.ppb;
  }
  if (g.dtype == RETRO_BF16)
    return g.D == 128 ? score_d<bf16_t, 128>(g, step, q_cur, q_batch_stride, c, k_new, v_new, scores, sa, s)
                      : score_d<bf16_t, 64>(g, step, q_cur, q_batch_stride, c, k_new, v_new, scores, sa, s);
  return g.D == 128 ? score_d<float, 128>(g, step, q_cur, q_batch_stride, c, k_new, v_new, scores, sa, s)
                    : score_d<float, 64>(g, step, q_cur, q_batch_stride, c, k_new, v_new, scores, sa, s);
}

}  // namespace retro
