// KV storage: AppendKV (Alg. 1) and bulk prefill, keeping the Quest page digests
// (element-wise key min / max of each page, Sec. 2.1) and, on append, the
// retrospective-mask override of Alg. 2's current-page rule.
#include <algorithm>

#include "internal.h"

namespace retro {
namespace {

template <typename T>
__device__ __forceinline__ bool less(T a, T b) { return to_f32(a) < to_f32(b); }

// One workgroup per sequence.  The token's keys / values and the digest row of
// its logical page are fetched together with the page-table entry (the digest is
// indexed by logical page, so it does not wait for the lookup).  Every thread
// reads seq_lens[b] before thread 0 advances it.
template <typename T>
__global__ void __launch_bounds__(256) append_kernel(Geometry g, int step, T* __restrict__ kc,
                                                     T* __restrict__ vc, T* __restrict__ dg,
                                                     const int32_t* __restrict__ pt,
                                                     int32_t* __restrict__ seq_lens,
                                                     int32_t* __restrict__ A,
                                                     const T* __restrict__ k_new,
                                                     const T* __restrict__ v_new) {
  constexpr int kPer = 8;
  const int b = blockIdx.x;
  const int n = g.hk * g.D;
  const int pos = seq_lens[b];
  const int lp = pos / g.P, slot = pos - lp * g.P;
  const bool lp_ok = pos >= 0 && lp < g.max_pages;
  int phys = -1;
  if (lp_ok) phys = pt[(int64_t)b * g.max_pages + lp];
  for (int base = 0; base < n; base += kPer * blockDim.x) {
    T kv[kPer], vv[kPer], lo[kPer], hi[kPer];
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int e = base + threadIdx.x + j * blockDim.x;
      if (e < n && lp_ok) {
        const int h = e / g.D, i = e - h * g.D;
        kv[j] = k_new[(int64_t)b * n + e];
        vv[j] = v_new[(int64_t)b * n + e];
        const T* d = dg + ((((int64_t)b * g.hk + h) * g.max_pages + lp) * 2) * g.D + i;
        if (slot != 0) {
          lo[j] = d[0];
          hi[j] = d[g.D];
        }
      }
    }
    const bool ok = lp_ok && phys >= 0 && phys < g.num_phys;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int e = base + threadIdx.x + j * blockDim.x;
      if (e >= n || !ok) continue;
      const int h = e / g.D, i = e - h * g.D;
      const int64_t ph = (int64_t)phys * g.hk + h;
      kc[(ph * g.P + slot) * g.D + i] = kv[j];
      vc[(ph * g.D + i) * g.P + slot] = vv[j];
      T* d = dg + ((((int64_t)b * g.hk + h) * g.max_pages + lp) * 2) * g.D + i;
      if (slot == 0) {
        d[0] = kv[j];
        d[g.D] = kv[j];
      } else {
        if (less(kv[j], lo[j])) d[0] = kv[j];
        if (less(hi[j], kv[j])) d[g.D] = kv[j];
      }
    }
  }
  const bool ok = lp_ok && phys >= 0 && phys < g.num_phys;
  if (ok)
    for (int h = threadIdx.x; h < g.hk; h += blockDim.x)
      A[((int64_t)b * g.hk + h) * g.max_pages + lp] = step - 1;
  __syncthreads();
  if (ok && threadIdx.x == 0) seq_lens[b] = pos + 1;
}

// Several tokens per sequence in one launch (AppendKV of Alg. 1 applied to
// tokens 0, 1, ..., n_tok - 1 in order, as n_tok calls of the one-token append
// would): token j goes to position seq_lens[b] + j.  One workgroup per
// sequence, one thread per (KV head, element) of a token.  The page-table
// entries of the pages the call touches are read once, in parallel, into LDS;
// the first token whose page is not mapped (or lies past max_pages) is dropped
// and so is every token after it (each would target the same position), as
// with the one-token append.  Each thread reads the keys and values of up to
// kChunk tokens before storing any, and the stored digest of the first page
// (whose first new slot may be past 0) alongside.
constexpr int kAppendMaxTokens = 64;   // tokens per launch (the host splits longer calls)
constexpr int kAppendThreads = 1024;

template <typename T>
__global__ void __launch_bounds__(kAppendThreads) append_tokens_kernel(
    Geometry g, int step, int n_tok, T* __restrict__ kc, T* __restrict__ vc, T* __restrict__ dg,
    const int32_t* __restrict__ pt, int32_t* __restrict__ seq_lens, int32_t* __restrict__ A,
    const T* __restrict__ k_new, const T* __restrict__ v_new) {
  constexpr int kChunk = 8;
  __shared__ int s_phys[kAppendMaxTokens + 1];
  __shared__ int s_nok;
  const int b = blockIdx.x;
  const int n = g.hk * g.D;
  const int pos0 = seq_lens[b];
  const int lp0 = pos0 >= 0 ? pos0 / g.P : 0;
  const int npages = pos0 >= 0 ? (pos0 + n_tok - 1) / g.P - lp0 + 1 : 0;
  if (threadIdx.x == 0) s_nok = pos0 >= 0 ? n_tok : 0;
  __syncthreads();
  if ((int)threadIdx.x < npages) {
    const int lp = lp0 + (int)threadIdx.x;
    const int ph = lp < g.max_pages ? pt[(int64_t)b * g.max_pages + lp] : -1;
    const bool ok = ph >= 0 && ph < g.num_phys;
    s_phys[threadIdx.x] = ok ? ph : -1;
    if (!ok) atomicMin(&s_nok, max(lp * g.P - pos0, 0));
  }
  __syncthreads();
  const int n_ok = s_nok;
  const int slot0 = pos0 - lp0 * g.P;
  for (int e = threadIdx.x; e < n && n_ok > 0; e += blockDim.x) {
    const int h = e / g.D, i = e - h * g.D;
    T* d = dg + ((((int64_t)b * g.hk + h) * g.max_pages + lp0) * 2) * g.D + i;
    T lo{}, hi{};
    if (slot0 != 0) {  // the first page already holds keys: widen its digest
      lo = d[0];
      hi = d[g.D];
    }
    int lp_cur = lp0;
    for (int j0 = 0; j0 < n_ok; j0 += kChunk) {
      T kv[kChunk], vv[kChunk];
#pragma unroll
      for (int jj = 0; jj < kChunk; ++jj) {
        const int j = min(j0 + jj, n_ok - 1);
        const int64_t src = ((int64_t)j * g.batch + b) * n + e;  // [token][batch][h_k][d]
        kv[jj] = k_new[src];
        vv[jj] = v_new[src];
      }
#pragma unroll
      for (int jj = 0; jj < kChunk; ++jj) {
        const int j = j0 + jj;
        if (j >= n_ok) break;
        const int pos = pos0 + j, lp = pos / g.P, slot = pos - lp * g.P;
        if (lp != lp_cur) {  // the previous page is complete: its digest goes out
          d[0] = lo;
          d[g.D] = hi;
          lp_cur = lp;
          d = dg + ((((int64_t)b * g.hk + h) * g.max_pages + lp) * 2) * g.D + i;
        }
        const int64_t ph = (int64_t)s_phys[lp - lp0] * g.hk + h;
        kc[(ph * g.P + slot) * g.D + i] = kv[jj];
        vc[(ph * g.D + i) * g.P + slot] = vv[jj];
        if (slot == 0) {
          lo = kv[jj];
          hi = kv[jj];
        } else {
          if (less(kv[jj], lo)) lo = kv[jj];
          if (less(hi, kv[jj])) hi = kv[jj];
        }
      }
    }
    d[0] = lo;
    d[g.D] = hi;
  }
  // Alg. 2's current-page rule for every page that received a key, every head
  if (n_ok > 0) {
    const int nlp = (pos0 + n_ok - 1) / g.P - lp0 + 1;
    for (int x = threadIdx.x; x < nlp * g.hk; x += blockDim.x) {
      const int h = x % g.hk, lp = lp0 + x / g.hk;
      A[((int64_t)b * g.hk + h) * g.max_pages + lp] = step - 1;
    }
  }
  __syncthreads();  // every thread has read seq_lens[b]
  if (n_ok > 0 && threadIdx.x == 0) seq_lens[b] = pos0 + n_ok;
}

// Prefill, pass 1: one workgroup per token copies its keys (token-major page) and
// values (d-major page).
template <typename T>
__global__ void __launch_bounds__(256) prefill_write_kernel(Geometry g, int seq, int start,
                                                            T* __restrict__ kc,
                                                            T* __restrict__ vc,
                                                            const int32_t* __restrict__ pt,
                                                            const T* __restrict__ k_src,
                                                            const T* __restrict__ v_src) {
  const int j = blockIdx.x;
  const int pos = start + j;
  const int lp = pos / g.P, slot = pos - lp * g.P;
  if (lp >= g.max_pages) return;
  const int phys = pt[(int64_t)seq * g.max_pages + lp];
  if (phys < 0 || phys >= g.num_phys) return;
  const int n = g.hk * g.D;
  for (int e = threadIdx.x; e < n; e += blockDim.x) {
    const int h = e / g.D, i = e - h * g.D;
    const int64_t ph = (int64_t)phys * g.hk + h;
    kc[(ph * g.P + slot) * g.D + i] = k_src[(int64_t)j * n + e];
    vc[(ph * g.D + i) * g.P + slot] = v_src[(int64_t)j * n + e];
  }
}

// Prefill, pass 2: digest of every touched page = min / max over its stored slots.
template <typename T>
__global__ void __launch_bounds__(128) prefill_digest_kernel(Geometry g, int seq, int start,
                                                             int end, const T* __restrict__ kc,
                                                             T* __restrict__ dg,
                                                             const int32_t* __restrict__ pt,
                                                             int32_t* __restrict__ seq_lens) {
  const int lp = start / g.P + blockIdx.x;
  const int h = blockIdx.y;
  if (blockIdx.x == 0 && h == 0 && threadIdx.x == 0) seq_lens[seq] = end;
  if (lp >= g.max_pages) return;
  const int phys = pt[(int64_t)seq * g.max_pages + lp];
  if (phys < 0 || phys >= g.num_phys) return;
  const int filled = min(g.P, end - lp * g.P);
  const int64_t ph = (int64_t)phys * g.hk + h;
  T* drow = dg + ((((int64_t)seq * g.hk + h) * g.max_pages + lp) * 2) * g.D;
  for (int i = threadIdx.x; i < g.D; i += blockDim.x) {
    T lo = kc[(ph * g.P) * g.D + i], hi = lo;
    for (int s = 1; s < filled; ++s) {
      const T v = kc[(ph * g.P + s) * g.D + i];
      if (less(v, lo)) lo = v;
      if (less(hi, v)) hi = v;
    }
    drow[i] = lo;
    drow[g.D + i] = hi;
  }
}

// UpdateKV (Alg. 1; Sec. 3.3, retrospective KV cache update): the n most recent
// stored tokens of every sequence are overwritten with their re-embedded keys and
// values, and the digest of each page they touch is recomputed from the page's
// stored keys (a min / max cannot be narrowed incrementally).  One workgroup per
// (touched page, KV head, sequence), one thread per element of d: each slot's key
// is the update when its position is in the updated run, else the stored one;
// all of a page's loads are issued before the min / max chain uses them.
__device__ __forceinline__ float key_f32(float x) { return x; }
__device__ __forceinline__ float key_f32(bf16_t x) { return to_f32(x); }
__device__ __forceinline__ void from_key(float x, float* d) { *d = x; }
__device__ __forceinline__ void from_key(float x, bf16_t* d) {
  d->bits = (uint16_t)(__float_as_uint(x) >> 16);  // exact: x holds a bf16 value
}

template <typename T, int PS>
__global__ void __launch_bounds__(128) update_kv_kernel(Geometry g, int n, T* __restrict__ kc,
                                                        T* __restrict__ vc, T* __restrict__ dg,
                                                        const int32_t* __restrict__ pt,
                                                        const int32_t* __restrict__ seq_lens,
                                                        const T* __restrict__ k_upd,
                                                        const T* __restrict__ v_upd) {
  const int b = blockIdx.z, h = blockIdx.y;
  const int len = seq_lens[b];
  const int start = max(len - n, 0);
  const int lp = start / PS + blockIdx.x;
  if (lp >= g.max_pages || lp * PS >= len) return;
  const int phys = pt[(int64_t)b * g.max_pages + lp];
  if (phys < 0 || phys >= g.num_phys) return;
  const int filled = min(PS, len - lp * PS);
  const int64_t ph = (int64_t)phys * g.hk + h;
  T* drow = dg + ((((int64_t)b * g.hk + h) * g.max_pages + lp) * 2) * g.D;
  for (int i = threadIdx.x; i < g.D; i += blockDim.x) {
    float f[PS];
#pragma unroll
    for (int s = 0; s < PS; ++s) {
      const int pos = lp * PS + s;
      if (s < filled) {  // uniform
        if (pos >= start) {
          const int64_t e = (((int64_t)b * n + (pos - (len - n))) * g.hk + h) * g.D + i;
          const T kv = k_upd[e];
          kc[(ph * PS + s) * g.D + i] = kv;
          vc[(ph * g.D + i) * PS + s] = v_upd[e];
          f[s] = key_f32(kv);
        } else {
          f[s] = key_f32(kc[(ph * PS + s) * g.D + i]);
        }
      }
    }
    float lo = f[0], hi = f[0];
#pragma unroll
    for (int s = 1; s < PS; ++s) {
      if (s < filled) {
        if (f[s] < lo) lo = f[s];
        if (hi < f[s]) hi = f[s];
      }
    }
    from_key(lo, drow + i);
    from_key(hi, drow + g.D + i);
  }
}

template <typename T>
hipError_t update_kv_t(const Geometry& g, const retro_kv_cache& c, int n, const void* k_upd,
                       const void* v_upd, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  // the run [len - n, len) spans at most ceil(n / P) + 1 pages
  const dim3 grid((unsigned)((n + g.P - 1) / g.P + 1), (unsigned)g.hk, (unsigned)g.batch);
  if (g.P == 16)
    update_kv_kernel<T, 16><<<grid, 128, 0, s>>>(g, n, (T*)c.k_cache, (T*)c.v_cache, (T*)c.digest,
                                                 c.page_table, c.seq_lens, (const T*)k_upd,
                                                 (const T*)v_upd);
  else
    update_kv_kernel<T, 32><<<grid, 128, 0, s>>>(g, n, (T*)c.k_cache, (T*)c.v_cache, (T*)c.digest,
                                                 c.page_table, c.seq_lens, (const T*)k_upd,
                                                 (const T*)v_upd);
  return hipGetLastError();
}

template <typename T>
hipError_t append_t(const Geometry& g, int step, const retro_kv_cache& c, const void* k_new,
                    const void* v_new, hipStream_t s) {
  append_kernel<T><<<g.batch, 256, 0, s>>>(g, step, (T*)c.k_cache, (T*)c.v_cache, (T*)c.digest,
                                           c.page_table, c.seq_lens, c.last_loaded,
                                           (const T*)k_new, (const T*)v_new);
  return hipGetLastError();
}

template <typename T>
hipError_t append_tokens_t(const Geometry& g, int step, const retro_kv_cache& c, int n_tok,
                           const void* k_new, const void* v_new, hipStream_t s) {
  const size_t tok_elems = (size_t)g.batch * g.hk * g.D;
  for (int j0 = 0; j0 < n_tok; j0 += kAppendMaxTokens) {
    const int nt = std::min(kAppendMaxTokens, n_tok - j0);
    append_tokens_kernel<T><<<g.batch, kAppendThreads, 0, s>>>(
        g, step, nt, (T*)c.k_cache, (T*)c.v_cache, (T*)c.digest, c.page_table, c.seq_lens,
        c.last_loaded, (const T*)k_new + j0 * tok_elems, (const T*)v_new + j0 * tok_elems);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

template <typename T>
hipError_t prefill_t(const Geometry& g, const retro_kv_cache& c, int seq, int start, int n,
                     const void* k_src, const void* v_src, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  prefill_write_kernel<T><<<n, 256, 0, s>>>(g, seq, start, (T*)c.k_cache, (T*)c.v_cache,
                                            c.page_table, (const T*)k_src, (const T*)v_src);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int end = start + n;
  const int pages = (end - 1) / g.P - start / g.P + 1;
  prefill_digest_kernel<T><<<dim3(pages, g.hk), 128, 0, s>>>(g, seq, start, end,
                                                             (const T*)c.k_cache,
                                                             (T*)c.digest, c.page_table,
                                                             c.seq_lens);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_append(const Geometry& g, int step, const retro_kv_cache& c, const void* k_new,
                         const void* v_new, hipStream_t s) {
  return g.dtype == RETRO_BF16 ? append_t<bf16_t>(g, step, c, k_new, v_new, s)
                               : append_t<float>(g, step, c, k_new, v_new, s);
}

hipError_t launch_append_tokens(const Geometry& g, int step, const retro_kv_cache& c, int n_tok,
                                const void* k_new, const void* v_new, hipStream_t s) {
  return g.dtype == RETRO_BF16 ? append_tokens_t<bf16_t>(g, step, c, n_tok, k_new, v_new, s)
                               : append_tokens_t<float>(g, step, c, n_tok, k_new, v_new, s);
}

hipError_t launch_prefill(const Geometry& g, const retro_kv_cache& c, int seq, int start, int n,
                          const void* k_src, const void* v_src, hipStream_t s) {
  return g.dtype == RETRO_BF16 ? prefill_t<bf16_t>(g, c, seq, start, n, k_src, v_src, s)
                               : prefill_t<float>(g, c, seq, start, n, k_src, v_src, s);
}

hipError_t launch_update_kv(const Geometry& g, const retro_kv_cache& c, int n, const void* k_upd,
                            const void* v_upd, hipStream_t s) {
  return g.dtype == RETRO_BF16 ? update_kv_t<bf16_t>(g, c, n, k_upd, v_upd, s)
                               : update_kv_t<float>(g, c, n, k_upd, v_upd, s);
}

}  // namespace retro
