// PageSelect + UpdateAndBuildMask (Alg. 1, Alg. 2) for one (sequence, KV head) per
// workgroup.
//
// 1. Page i of the sequence belongs to thread i mod THREADS (stripe i /
//    THREADS), so every load is coalesced.  Page-table entries, last_loaded
//    values and scores (mapped to order-preserving 32-bit keys: larger float ->
//    larger key, -0 == +0) are all requested before any is used.
// 2. Radix select over rel = key - min_key with 11-bit digits taken from the
//    top of rel's actual bit length.  Each pass histograms the digit of the
//    keys still in the running into a histogram of its own (so none is cleared
//    between passes); one wavefront scans it (a prefix sum over its lanes' bin
//    totals locates T, the k-th largest key) and publishes T's digit through
//    LDS, and `need` becomes the number of keys to take from T's bin.  The
//    search stops as soon as that bin is taken whole or all bits are fixed;
//    a bin of at most 64 keys is instead listed in LDS and ranked exactly by
//    one wavefront.
// 3. Compaction in page order: a page is kept if its rel is above T's prefix,
//    or ties with it and is among the first `need` such pages (ties go to the
//    lower page index).  Ballots count kept pages below a lane within its
//    wavefront and stripe; one scan over the (stripe, wavefront) table, which
//    is in page order, adds the pages below in other wavefronts and stripes.
// 4. Alg. 2 for the kept pages: mask = last_loaded[p]; last_loaded[p] = step.
//    Kept pages are distinct, so each thread updates its own.  The physical page
//    of every kept page is written too (for the attention kernel).
#include "roles.h"

namespace retro {
namespace {

template <int THREADS, int PER>
__global__ void __launch_bounds__(THREADS) topk_mask_kernel(TopkArgs ta,
                                                            const int32_t* __restrict__ seq_lens) {
  __shared__ __attribute__((aligned(16))) uint32_t hist[kTopkHistWords];
  __shared__ int small[kTopkSmall];
  const int bh = blockIdx.x;
  const int b = bh / ta.g.hk;
  // a pending token (Geometry::token_pending) gets Alg. 2's current-page rule here
  int tok_lp = -1;
  if (ta.g.token_pending) {
    const int pos = seq_lens[b];
    if (token_phys(ta.g, ta.pt, b, pos) >= 0) tok_lp = pos / ta.g.P;
  }
  topk_role<PER, THREADS / 64, false>(
      ta, bh,
      [&] { return live_seq_len(ta.g, seq_lens, ta.pt, b); },
      tok_lp, hist, small, [] {});
}

// Alg. 2 on the kept selection of a top-k reuse step: one wavefront per
// (sequence, KV head); every mask value is read before any last_loaded entry
// of the head changes (the rows hold distinct pages).
__global__ void __launch_bounds__(64) reuse_mask_kernel(Geometry g, int step,
                                                        const int32_t* __restrict__ sel,
                                                        int32_t* __restrict__ msk,
                                                        const int32_t* __restrict__ nsel,
                                                        int32_t* __restrict__ A) {
  const int bh = blockIdx.x;
  const int k = min(max(nsel[bh], 0), g.k_max);
  const int32_t* row = sel + (int64_t)bh * g.k_max;
  int32_t* m = msk + (int64_t)bh * g.k_max;
  int32_t* a = A + (int64_t)bh * g.max_pages;
  for (int i = threadIdx.x; i < g.k_max; i += 64) {
    const int p = i < k ? row[i] : -1;
    m[i] = (p >= 0 && p < g.max_pages) ? a[p] : -1;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < k; i += 64) {
    const int p = row[i];
    if (p >= 0 && p < g.max_pages) a[p] = step;
  }
}

}  // namespace

bool reuse_step(const Geometry& g, int step) { return g.reuse >= 2 && step % g.reuse != 0; }

hipError_t launch_reuse_mask(const Geometry& g, int step, const retro_kv_cache& c,
                             const retro_selection& sel, hipStream_t s) {
  reuse_mask_kernel<<<(unsigned)(g.batch * g.hk), 64, 0, s>>>(g, step, sel.selected, sel.mask,
                                                             sel.num_selected, c.last_loaded);
  return hipGetLastError();
}

hipError_t launch_topk_mask(const Geometry& g, int step, const float* scores,
                            const retro_kv_cache& c, const retro_selection& sel,
                            int32_t* sel_phys, hipStream_t s) {
  TopkArgs ta{g, step, scores, c.page_table, c.last_loaded, sel.selected, sel.mask,
              sel.num_selected, sel_phys};
  const unsigned grid = (unsigned)(g.batch * g.hk);
  // one workgroup per head: its time is one wavefront's instruction count,
  // so sixteen wavefronts share the pages
  if (g.max_pages <= 1024 * 3)
    topk_mask_kernel<1024, 3><<<grid, 1024, 0, s>>>(ta, c.seq_lens);
  else if (g.max_pages <= 1024 * 6)
    topk_mask_kernel<1024, 6><<<grid, 1024, 0, s>>>(ta, c.seq_lens);
  else
    topk_mask_kernel<1024, 16><<<grid, 1024, 0, s>>>(ta, c.seq_lens);
  return hipGetLastError();
}

}  // namespace retro
