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
#include "internal.h"

namespace retro {
namespace {

__device__ __forceinline__ uint32_t order_key(float s) {
  uint32_t u = __float_as_uint(s);
  if (u == 0x80000000u) u = 0u;  // -0 ranks as +0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Exclusive prefix sum over the workgroup.
template <int NW>
__device__ __forceinline__ int block_exclusive_scan(int v, int* sh) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) sh[wave] = x;
  __syncthreads();
  int off = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w)
    if (w < wave) off += sh[w];
  __syncthreads();
  return off + x - v;
}

template <int THREADS, int PER>
__global__ void __launch_bounds__(THREADS) topk_mask_kernel(Geometry g, int step,
                                                            const float* __restrict__ scores,
                                                            const int32_t* __restrict__ seq_lens,
                                                            const int32_t* __restrict__ pt,
                                                            int32_t* __restrict__ A,
                                                            int32_t* __restrict__ selected,
                                                            int32_t* __restrict__ mask,
                                                            int32_t* __restrict__ num_selected,
                                                            int32_t* __restrict__ sel_phys) {
  constexpr int NW = THREADS / 64;
  constexpr int NB = 2048;             // bins of an 11-bit digit
  constexpr int BPT = NB / THREADS;    // bins per thread in the suffix scan
  __shared__ uint32_t hist[NB];
  __shared__ int scan_sh[NW];
  __shared__ uint32_t red_sh[2 * NW];
  __shared__ uint32_t s_digit, s_above, s_count;

  const int bh = blockIdx.x;
  const int b = bh / g.hk;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int per = (g.max_pages + THREADS - 1) / THREADS;
  const int base = tid * per;
  const float* srow = scores + (int64_t)bh * g.max_pages;
  int32_t* a_row = A + (int64_t)bh * g.max_pages;
  const int32_t* p_row = pt + (int64_t)b * g.max_pages;

  uint32_t key[PER];
  int32_t a_old[PER], phys[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int idx = base + j;
    if (j < per && idx < g.max_pages) {
      key[j] = order_key(srow[idx]);
      a_old[j] = a_row[idx];
      phys[j] = p_row[idx];
    } else {
      key[j] = 0u;
      a_old[j] = -1;
      phys[j] = -1;
    }
  }
  const int n = min((seq_lens[b] + g.P - 1) / g.P, g.max_pages);
  const int k = min(g.budget / g.P, n);
  auto valid = [&](int j) { return j < per && base + j < n; };

  // rel = key - kmin over the valid keys; T is searched among rel values.
  uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
#pragma unroll
  for (int j = 0; j < PER; ++j)
    if (valid(j)) {
      kmin = min(kmin, key[j]);
      kmax = max(kmax, key[j]);
    }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    kmin = min(kmin, (uint32_t)__shfl_xor((int)kmin, m));
    kmax = max(kmax, (uint32_t)__shfl_xor((int)kmax, m));
  }
  if (lane == 0) {
    red_sh[wave] = kmin;
    red_sh[NW + wave] = kmax;
  }
  __syncthreads();
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    kmin = min(kmin, red_sh[w]);
    kmax = max(kmax, red_sh[NW + w]);
  }
  const uint32_t range = kmax - kmin;
  const int nbits = range ? 32 - __clz((int)range) : 1;
  uint64_t prefix = 0u;  // chosen digits of T's rel, bits [lo, nbits)
  int lo = nbits;
  int need = k;
  if (k > 0 && k < n) {
#pragma unroll 1
    for (int hi = nbits; hi > 0; hi = lo) {
      lo = max(hi - 11, 0);
      const uint32_t dmask = (1u << (hi - lo)) - 1u;
      for (int i = tid; i < NB; i += THREADS) hist[i] = 0u;
      __syncthreads();
#pragma unroll
      for (int j = 0; j < PER; ++j) {
        const uint64_t rel = key[j] - kmin;
        if (valid(j) && (rel >> hi) == prefix) atomicAdd(&hist[(rel >> lo) & dmask], 1u);
      }
      __syncthreads();
      // suffix scan: thread t owns bins [NB - BPT*(t+1), NB - BPT*t), descending
      uint32_t local = 0u;
#pragma unroll
      for (int i = 0; i < BPT; ++i) local += hist[NB - 1 - (tid * BPT + i)];
      uint32_t cum = (uint32_t)block_exclusive_scan<NW>((int)local, scan_sh);
#pragma unroll
      for (int i = 0; i < BPT; ++i) {
        const int bin = NB - 1 - (tid * BPT + i);
        const uint32_t c = hist[bin];
        if (cum < (uint32_t)need && cum + c >= (uint32_t)need) {
          s_digit = (uint32_t)bin;
          s_above = cum;
          s_count = c;
        }
        cum += c;
      }
      __syncthreads();
      need -= (int)s_above;
      prefix = (prefix << (hi - lo)) | s_digit;
      if ((int)s_count == need) break;  // the whole bin is kept: T's prefix suffices
    }
  }
  // compaction in page order
  int c_eq = 0;
#pragma unroll
  for (int j = 0; j < PER; ++j)
    if (valid(j) && ((uint64_t)(key[j] - kmin) >> lo) == prefix) ++c_eq;
  const int eq_before = block_exclusive_scan<NW>(c_eq, scan_sh);
  uint32_t take = 0u;
  int n_take = 0, eq_seen = 0;
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    bool t = false;
    if (valid(j)) {
      if (k >= n) {
        t = true;
      } else if (k > 0) {
        const uint64_t km = (uint64_t)(key[j] - kmin) >> lo;
        if (km > prefix) {
          t = true;
        } else if (km == prefix) {
          t = (eq_before + eq_seen) < need;
          ++eq_seen;
        }
      }
    }
    take |= (t ? 1u : 0u) << j;
    n_take += t ? 1 : 0;
  }
  int pos = block_exclusive_scan<NW>(n_take, scan_sh);
  int32_t* sel_row = selected + (int64_t)bh * g.k_max;
  int32_t* m_row = mask + (int64_t)bh * g.k_max;
  int32_t* ph_row = sel_phys ? sel_phys + (int64_t)bh * g.k_max : nullptr;
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    if (take & (1u << j)) {
      const int p = base + j;
      sel_row[pos] = p;
      m_row[pos] = a_old[j];
      a_row[p] = step;
      if (ph_row) ph_row[pos] = (phys[j] >= 0 && phys[j] < g.num_phys) ? phys[j] : -1;
      ++pos;
    }
  }
  for (int i = k + tid; i < g.k_max; i += THREADS) {
    sel_row[i] = -1;
    m_row[i] = -1;
    if (ph_row) ph_row[i] = -1;
  }
  if (tid == 0) num_selected[bh] = k;
}

}  // namespace

hipError_t launch_topk_mask(const Geometry& g, int step, const float* scores,
                            const retro_kv_cache& c, const retro_selection& sel,
                            int32_t* sel_phys, hipStream_t s) {
  if (g.max_pages <= 256 * 24) {
    topk_mask_kernel<256, 24><<<g.batch * g.hk, 256, 0, s>>>(
        g, step, scores, c.seq_lens, c.page_table, c.last_loaded, sel.selected, sel.mask,
        sel.num_selected, sel_phys);
  } else {
    topk_mask_kernel<1024, 16><<<g.batch * g.hk, 1024, 0, s>>>(
        g, step, scores, c.seq_lens, c.page_table, c.last_loaded, sel.selected, sel.mask,
        sel.num_selected, sel_phys);
  }
  return hipGetLastError();
}

}  // namespace retro
