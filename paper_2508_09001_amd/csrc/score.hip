// Page criticality score, eq. (quest_score), per (sequence, KV head, page):
//   score = sum over the G query heads g of the KV head of
//           sum_i max(q_gi * Kmin_i, q_gi * Kmax_i)
// evaluated in fp32 in one fixed order so that page selection is exact:
// products rounded to fp32, the d terms summed as a perfect binary tree over
// index order (pairwise summation), the per-head sums added in head order, and
// + 0.0f at the end.
//
// Layout of the work: digests are stored per logical page, so a KV head's
// digests form one contiguous stream.  A page's digest row (d elements of Kmin,
// then d of Kmax) is read as 16-byte vectors by LPP = d / VEC consecutive lanes,
// lane c holding elements [c*VEC, (c+1)*VEC).  The tree's first log2(VEC) levels are in-lane,
// the remaining log2(LPP) levels pair neighbouring lanes (xor 1, 2, 4, ...), so
// the order is the pairwise order over all d terms.  A wavefront covers
// 64 / LPP pages per iteration; a workgroup of four wavefronts scores a block
// of consecutive logical pages of one (sequence, KV head).
#include "internal.h"

namespace retro {
namespace {

constexpr int kScoreIters = 4;

template <typename T>
__device__ __forceinline__ void unpack(const uint4& u, float* out);

template <>
__device__ __forceinline__ void unpack<bf16_t>(const uint4& u, float* out) {
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    out[2 * i] = __uint_as_float(w[i] << 16);
    out[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
  }
}

template <>
__device__ __forceinline__ void unpack<float>(const uint4& u, float* out) {
  out[0] = __uint_as_float(u.x);
  out[1] = __uint_as_float(u.y);
  out[2] = __uint_as_float(u.z);
  out[3] = __uint_as_float(u.w);
}

template <typename T, int D>
__global__ void __launch_bounds__(256) score_kernel(Geometry g, const T* __restrict__ q,
                                                   int64_t q_bstride, const T* __restrict__ dg,
                                                   const int32_t* __restrict__ seq_lens,
                                                   float* __restrict__ scores) {
#pragma clang fp contract(off)
  constexpr int VEC = 16 / sizeof(T);
  constexpr int LPP = D / VEC;
  constexpr int PPW = 64 / LPP;
  constexpr int PPB = 4 * PPW * kScoreIters;
  extern __shared__ float sq[];  // [G][D] the group's current queries, as fp32

  const int b = blockIdx.z, h = blockIdx.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = lane % LPP;
  // Every load of the block is issued before any is waited on: the digest rows
  // (in bounds of the [max_pages] row whatever the sequence length), the queries
  // and the sequence length.
  const T* drow = dg + ((int64_t)b * g.hk + h) * g.max_pages * 2 * D;
  uint4 raw[kScoreIters][2];
#pragma unroll
  for (int it = 0; it < kScoreIters; ++it) {
    const int page = blockIdx.x * PPB + (wave * kScoreIters + it) * PPW + lane / LPP;
    if (page < g.max_pages) {
      const T* row = drow + (int64_t)page * 2 * D + c * VEC;
      raw[it][0] = *reinterpret_cast<const uint4*>(row);
      raw[it][1] = *reinterpret_cast<const uint4*>(row + D);
    } else {
      raw[it][0] = raw[it][1] = make_uint4(0u, 0u, 0u, 0u);
    }
  }
  const T* qb = q + (int64_t)b * q_bstride + (int64_t)h * g.G * D;
  for (int e = threadIdx.x; e < g.G * D; e += blockDim.x) sq[e] = to_f32(qb[e]);
  const int n_pages = min((seq_lens[b] + g.P - 1) / g.P, g.max_pages);
  __syncthreads();

#pragma unroll
  for (int it = 0; it < kScoreIters; ++it) {
    const int page = blockIdx.x * PPB + (wave * kScoreIters + it) * PPW + lane / LPP;
    float lo[VEC], hi[VEC];
    unpack<T>(raw[it][0], lo);
    unpack<T>(raw[it][1], hi);
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
    if (page < n_pages && c == 0) scores[((int64_t)b * g.hk + h) * g.max_pages + page] = S + 0.0f;
  }
}

template <typename T, int D>
hipError_t score_t(const Geometry& g, const void* q, int64_t qbs, const retro_kv_cache& c,
                   float* scores, hipStream_t s) {
  constexpr int VEC = 16 / sizeof(T);
  constexpr int PPB = 4 * (64 / (D / VEC)) * kScoreIters;
  dim3 grid((g.max_pages + PPB - 1) / PPB, g.hk, g.batch);
  const size_t lds = sizeof(float) * g.G * D;
  score_kernel<T, D><<<grid, 256, lds, s>>>(g, (const T*)q, qbs, (const T*)c.digest, c.seq_lens,
                                             scores);
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
