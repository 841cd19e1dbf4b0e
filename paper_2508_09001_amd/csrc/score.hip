// Page criticality score, eq. (quest_score), per (sequence, KV head, page):
//   score = sum over the G query heads g of the KV head of
//           sum_i max(q_gi * Kmin_i, q_gi * Kmax_i)
// evaluated in fp32 in one fixed order so that page selection is exact:
// products rounded to fp32, the d terms summed as a perfect binary tree over
// index order (pairwise summation), the per-head sums added in head order, and
// + 0.0f at the end.
//
// Layout of the work: a page's digest row (d elements of Kmin, then d of Kmax)
// is read as 16-byte vectors by LPP = d / VEC consecutive lanes, lane c holding
// elements [c*VEC, (c+1)*VEC).  The tree's first log2(VEC) levels are in-lane,
// the remaining log2(LPP) levels pair neighbouring lanes (xor 1, 2, 4, ...), so
// the order is the pairwise order over all d terms.  A wavefront covers
// 64 / LPP pages per iteration; a workgroup of four wavefronts scores a block
// of consecutive logical pages of one (sequence, KV head).
#include "internal.h"

namespace retro {
namespace {

constexpr int kScoreIters = 4;

template <typename T>
__device__ __forceinline__ void load_vec(const T* p, float* out);

template <>
__device__ __forceinline__ void load_vec<bf16_t>(const bf16_t* p, float* out) {
  const uint4 u = *reinterpret_cast<const uint4*>(p);
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    out[2 * i] = __uint_as_float(w[i] << 16);
    out[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
  }
}

template <>
__device__ __forceinline__ void load_vec<float>(const float* p, float* out) {
  const float4 u = *reinterpret_cast<const float4*>(p);
  out[0] = u.x;
  out[1] = u.y;
  out[2] = u.z;
  out[3] = u.w;
}

template <typename T, int D>
__global__ void __launch_bounds__(256) score_kernel(Geometry g, const T* __restrict__ q,
                                                   int64_t q_bstride, const T* __restrict__ dg,
                                                   const int32_t* __restrict__ pt,
                                                   const int32_t* __restrict__ seq_lens,
                                                   float* __restrict__ scores) {
#pragma clang fp contract(off)
  constexpr int VEC = 16 / sizeof(T);
  constexpr int LPP = D / VEC;
  constexpr int PPW = 64 / LPP;
  constexpr int PPB = 4 * PPW * kScoreIters;
  extern __shared__ float sq[];  // [G][D] the group's current queries, as fp32

  const int b = blockIdx.z, h = blockIdx.y;
  const int n_pages = min((seq_lens[b] + g.P - 1) / g.P, g.max_pages);
  if ((int)blockIdx.x * PPB >= n_pages) return;  // uniform over the workgroup

  const T* qb = q + (int64_t)b * q_bstride + (int64_t)h * g.G * D;
  for (int e = threadIdx.x; e < g.G * D; e += blockDim.x) sq[e] = to_f32(qb[e]);
  __syncthreads();

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = lane % LPP;
#pragma unroll 1
  for (int it = 0; it < kScoreIters; ++it) {
    const int page = blockIdx.x * PPB + (wave * kScoreIters + it) * PPW + lane / LPP;
    const bool valid = page < n_pages;
    float lo[VEC], hi[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) lo[v] = hi[v] = 0.f;
    bool mapped = false;
    if (valid) {
      const int phys = pt[(int64_t)b * g.max_pages + page];
      if (phys >= 0 && phys < g.num_phys) {
        const T* row = dg + ((int64_t)phys * g.hk + h) * 2 * D + c * VEC;
        load_vec<T>(row, lo);
        load_vec<T>(row + D, hi);
        mapped = true;
      }
    }
    float S = 0.f;
    for (int gq = 0; gq < g.G; ++gq) {
      float t[VEC];
#pragma unroll
      for (int v = 0; v < VEC; ++v) {
        const float qv = sq[gq * D + c * VEC + v];
        const float a = qv * lo[v];
        const float b2 = qv * hi[v];
        t[v] = a > b2 ? a : b2;
      }
#pragma unroll
      for (int w = 1; w < VEC; w *= 2)
#pragma unroll
        for (int i = 0; i + w < VEC; i += 2 * w) t[i] = t[i] + t[i + w];
      float s = t[0];
#pragma unroll
      for (int m = 1; m < LPP; m *= 2) s = s + __shfl_xor(s, m);
      S = (gq == 0) ? s : S + s;
    }
    // An unmapped logical page (outside the caller's contract) holds no tokens:
    // it ranks below every real page.
    if (valid && c == 0)
      scores[((int64_t)b * g.hk + h) * g.max_pages + page] = mapped ? S + 0.0f : -INFINITY;
  }
}

template <typename T, int D>
hipError_t score_t(const Geometry& g, const void* q, int64_t qbs, const retro_kv_cache& c,
                   float* scores, hipStream_t s) {
  constexpr int VEC = 16 / sizeof(T);
  constexpr int PPB = 4 * (64 / (D / VEC)) * kScoreIters;
  dim3 grid((g.max_pages + PPB - 1) / PPB, g.hk, g.batch);
  const size_t lds = sizeof(float) * g.G * D;
  score_kernel<T, D><<<grid, 256, lds, s>>>(g, (const T*)q, qbs, (const T*)c.digest, c.page_table,
                                             c.seq_lens, scores);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_score(const Geometry& g, const void* q_cur, int64_t q_batch_stride,
                        const retro_kv_cache& c, float* scores, hipStream_t s) {
  if (g.dtype == RETRO_BF16)
    return g.D == 128 ? score_t<bf16_t, 128>(g, q_cur, q_batch_stride, c, scores, s)
                      : score_t<bf16_t, 64>(g, q_cur, q_batch_stride, c, scores, s);
  return g.D == 128 ? score_t<float, 128>(g, q_cur, q_batch_stride, c, scores, s)
                    : score_t<float, 64>(g, q_cur, q_batch_stride, c, scores, s);
}

}  // namespace retro
