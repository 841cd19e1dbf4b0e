// PageSelect + UpdateAndBuildMask (Alg. 1, Alg. 2) for one (sequence, KV head) per
// workgroup of 1024 threads.
//
// 1. Each thread holds a contiguous run of at most kPer page scores, mapped to
//    order-preserving 32-bit keys (larger float -> larger key, -0 == +0).
// 2. Radix select, most significant byte first (four passes of an LDS histogram
//    plus a suffix scan), finds T, the k-th largest key, and `need`, how many
//    keys equal to T belong to the top k.
// 3. Compaction in page order: a page is kept if its key is above T, or equal
//    to T and among the first `need` such pages (ties go to the lower page
//    index).  Two block-wide exclusive scans give each kept page its output slot,
//    so the output is in ascending page order.
// 4. Alg. 2 for the kept pages: mask = last_loaded[p]; last_loaded[p] = step.
//    Kept pages are distinct, so every thread updates its own pages.
#include "internal.h"

namespace retro {
namespace {

constexpr int kThreads = 1024;
constexpr int kPer = 16;  // pages per thread: max_pages <= 16384

__device__ __forceinline__ uint32_t order_key(float s) {
  uint32_t u = __float_as_uint(s);
  if (u == 0x80000000u) u = 0u;  // -0 ranks as +0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Exclusive prefix sum over the workgroup (1024 threads, 16 wavefronts).
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
  if (threadIdx.x < 64) {
    const int nw = blockDim.x >> 6;
    int w = threadIdx.x < nw ? sh[threadIdx.x] : 0;
    int incl = w;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(incl, o);
      if (threadIdx.x >= o) incl += y;
    }
    if (threadIdx.x < nw) sh[threadIdx.x] = incl - w;
  }
  __syncthreads();
  const int res = x - v + sh[wave];
  __syncthreads();
  return res;
}

__global__ void __launch_bounds__(kThreads) topk_mask_kernel(Geometry g, int step,
                                                             const float* __restrict__ scores,
                                                             const int32_t* __restrict__ seq_lens,
                                                             int32_t* __restrict__ A,
                                                             int32_t* __restrict__ selected,
                                                             int32_t* __restrict__ mask,
                                                             int32_t* __restrict__ num_selected) {
  __shared__ uint32_t hist[256];
  __shared__ int scan_sh[64];
  __shared__ uint32_t sel_digit, sel_above;

  const int bh = blockIdx.x;
  const int b = bh / g.hk;
  const int tid = threadIdx.x;
  const int n = min((seq_lens[b] + g.P - 1) / g.P, g.max_pages);
  const int k = min(g.budget / g.P, n);
  const int per = (n + kThreads - 1) / kThreads;
  const int base = tid * per;
  const float* srow = scores + (int64_t)bh * g.max_pages;

  uint32_t key[kPer];
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int idx = base + j;
    key[j] = (j < per && idx < n) ? order_key(srow[idx]) : 0u;
  }
  auto valid = [&](int j) { return j < per && base + j < n; };

  uint32_t T = 0u;
  int need = k;
  if (k > 0 && k < n) {
    uint32_t prefix = 0u, pmask = 0u;
#pragma unroll 1
    for (int pass = 0; pass < 4; ++pass) {
      const int shift = 24 - 8 * pass;
      if (tid < 256) hist[tid] = 0u;
      __syncthreads();
#pragma unroll
      for (int j = 0; j < kPer; ++j)
        if (valid(j) && (key[j] & pmask) == prefix) atomicAdd(&hist[(key[j] >> shift) & 255u], 1u);
      __syncthreads();
      // inclusive scan of hist[255], hist[254], ... gives suffix sums
      uint32_t hv = 0u, x = 0u;
      if (tid < 256) {
        const int lane = tid & 63;
        hv = hist[255 - tid];
        x = hv;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const uint32_t y = __shfl_up(x, o);
          if (lane >= o) x += y;
        }
        if (lane == 63) scan_sh[tid >> 6] = (int)x;
      }
      __syncthreads();
      if (tid < 256) {
        uint32_t off = 0u;
        for (int w = 0; w < (tid >> 6); ++w) off += (uint32_t)scan_sh[w];
        const uint32_t suffix = x + off;            // keys with digit >= 255 - tid
        const uint32_t above = suffix - hv;         // keys with digit >  255 - tid
        if (suffix >= (uint32_t)need && above < (uint32_t)need) {
          sel_digit = 255u - tid;
          sel_above = above;
        }
      }
      __syncthreads();
      need -= (int)sel_above;
      prefix |= sel_digit << shift;
      pmask |= 0xFFu << shift;
      __syncthreads();
    }
    T = prefix;
  }

  // compaction in page order
  int c_eq = 0;
#pragma unroll
  for (int j = 0; j < kPer; ++j)
    if (valid(j) && key[j] == T) ++c_eq;
  const int eq_before = block_exclusive_scan(c_eq, scan_sh);
  bool take[kPer];
  int n_take = 0, eq_seen = 0;
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    bool t = false;
    if (valid(j)) {
      if (k >= n) {
        t = true;
      } else if (k > 0) {
        if (key[j] > T) {
          t = true;
        } else if (key[j] == T) {
          t = (eq_before + eq_seen) < need;
          ++eq_seen;
        }
      }
    }
    take[j] = t;
    n_take += t ? 1 : 0;
  }
  int pos = block_exclusive_scan(n_take, scan_sh);
  int32_t* sel_row = selected + (int64_t)bh * g.k_max;
  int32_t* m_row = mask + (int64_t)bh * g.k_max;
  int32_t* a_row = A + (int64_t)bh * g.max_pages;
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    if (take[j]) {
      const int p = base + j;
      sel_row[pos] = p;
      m_row[pos] = a_row[p];
      a_row[p] = step;
      ++pos;
    }
  }
  for (int i = k + tid; i < g.k_max; i += kThreads) {
    sel_row[i] = -1;
    m_row[i] = -1;
  }
  if (tid == 0) num_selected[bh] = k;
}

}  // namespace

hipError_t launch_topk_mask(const Geometry& g, int step, const float* scores,
                            const retro_kv_cache& c, const retro_selection& sel, hipStream_t s) {
  topk_mask_kernel<<<g.batch * g.hk, kThreads, 0, s>>>(g, step, scores, c.seq_lens,
                                                        c.last_loaded, sel.selected, sel.mask,
                                                        sel.num_selected);
  return hipGetLastError();
}

}  // namespace retro
