// PageSelect + UpdateAndBuildMask (Alg. 1, Alg. 2) for one (sequence, KV head) per
// workgroup.
//
// 1. Each thread owns a contiguous run of logical pages and loads, all at once,
//    their scores (mapped to order-preserving 32-bit keys: larger float ->
//    larger key, -0 == +0), their last_loaded values and their page-table
//    entries.  Loads do not wait for the sequence length: runs are laid out over
//    the row's max_pages entries, which are all in bounds.
// 2. Radix select over rel = key - min_key, with 11-bit digits taken from the
//    top of rel's actual bit length (score keys span a narrow range, so even the
//    first digit spreads them over the 2048 bins and the LDS histogram atomics
//    rarely collide).  Each pass histograms the digit of the keys still in the
//    running, a suffix scan over the bins fixes the digit of T, the k-th
//    largest key, and `need` becomes the number of keys to take from T's bin.
//    The search stops as soon as that bin is taken whole or all bits are fixed.
// 3. Compaction in page order: a page is kept if its rel is above T's prefix,
//    or ties with it and is among the first `need` such pages (ties go to the
//    lower page index).  Two block-wide exclusive scans give each kept page its output slot,
//    so the output is in ascending page order.
// 4. Alg. 2 for the kept pages: mask = last_loaded[p]; last_loaded[p] = step.
//    Kept pages are distinct, so each thread updates its own.  The physical page
//    of every kept page is written too (for the attention kernel).
#include "roles.h"

namespace retro {
namespace {

template <int THREADS, int PER>
__global__ void __launch_bounds__(THREADS) topk_mask_kernel(TopkArgs ta,
                                                            const int32_t* __restrict__ seq_lens) {
  __shared__ uint32_t hist[kTopkBins];
  __shared__ int small[kTopkSmall];
  const int bh = blockIdx.x;
  const int b = bh / ta.g.hk;
  const int n = min((seq_lens[b] + ta.g.P - 1) / ta.g.P, ta.g.max_pages);
  topk_role<PER>(ta, bh, n, hist, small);
}

}  // namespace

hipError_t launch_topk_mask(const Geometry& g, int step, const float* scores,
                            const retro_kv_cache& c, const retro_selection& sel,
                            int32_t* sel_phys, hipStream_t s) {
  TopkArgs ta{g, step, scores, c.page_table, c.last_loaded, sel.selected, sel.mask,
              sel.num_selected, sel_phys};
  if (g.max_pages <= 256 * 24)
    topk_mask_kernel<256, 24><<<g.batch * g.hk, 256, 0, s>>>(ta, c.seq_lens);
  else
    topk_mask_kernel<1024, 16><<<g.batch * g.hk, 1024, 0, s>>>(ta, c.seq_lens);
  return hipGetLastError();
}

}  // namespace retro
