// Page criticality score, eq. (quest_score), per (sequence, KV head, page), in
// the fixed fp32 order described in roles.h (score_role).  Digests are stored
// per logical page, so a KV head's digests form one contiguous stream; a
// workgroup of four wavefronts scores a block of consecutive pages.
#include "roles.h"

namespace retro {
namespace {

constexpr int kScoreIters = 4;

template <typename T, int D>
__global__ void __launch_bounds__(256) score_kernel(Geometry g, const T* __restrict__ q,
                                                   int64_t q_bstride, T* __restrict__ dg,
                                                   const int32_t* __restrict__ seq_lens,
                                                   float* __restrict__ scores) {
  extern __shared__ float sq[];  // [G][D] the group's current queries, as fp32
  constexpr int PPB = 4 * ScoreShape<T, D>::PPW * kScoreIters;
  const int b = blockIdx.z, h = blockIdx.y;
  const int64_t bh = (int64_t)b * g.hk + h;
  const int n_pages = min((seq_lens[b] + g.P - 1) / g.P, g.max_pages);
  score_role<T, D, kScoreIters>(g, blockIdx.x * PPB, q + b * q_bstride + (int64_t)h * g.G * D,
                                dg + bh * g.max_pages * 2 * D, n_pages, scores + bh * g.max_pages,
                                sq, StepToken<T>{-1, 0, nullptr, nullptr, nullptr, nullptr, nullptr, 0});
}

template <typename T, int D>
hipError_t score_t(const Geometry& g, const void* q, int64_t qbs, const retro_kv_cache& c,
                   float* scores, hipStream_t s) {
  constexpr int PPB = 4 * ScoreShape<T, D>::PPW * kScoreIters;
  dim3 grid((g.max_pages + PPB - 1) / PPB, g.hk, g.batch);
  const size_t lds = sizeof(float) * g.G * D;
  score_kernel<T, D><<<grid, 256, lds, s>>>(g, (const T*)q, qbs, (T*)c.digest, c.seq_lens, scores);
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
