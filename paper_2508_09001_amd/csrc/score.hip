// Page criticality score, eq. (quest_score), per (sequence, KV head, page), in
// the fixed fp32 order described in roles.h (score_role).  Digests are stored
// per logical page, so a KV head's digests form one contiguous stream; a
// workgroup of four wavefronts scores a block of consecutive pages.
#include "roles.h"

namespace retro {
namespace {

// One pass of four pages per wavefront: many small workgroups keep several
// wavefronts per SIMD busy, which hides the dependent add chains of the tree.
constexpr int kScoreIters = 1;

struct TokenArgs {
  int step;
  const void* k_new;
  const void* v_new;
  void* kc;
  void* vc;
  const int32_t* pt;
  int32_t* A;
};

template <typename T, int D>
__global__ void __launch_bounds__(256) score_kernel(Geometry g, const T* __restrict__ q,
                                                   int64_t q_bstride, T* __restrict__ dg,
                                                   const int32_t* __restrict__ seq_lens,
                                                   float* __restrict__ scores, TokenArgs ta) {
  extern __shared__ float sq[];  // [G][D] the group's current queries, as fp32
  constexpr int PPB = 4 * ScoreShape<T, D>::PPW * kScoreIters;
  const int b = blockIdx.z, h = blockIdx.y;
  const int64_t bh = (int64_t)b * g.hk + h;
  const int pos = seq_lens[b];
  StepToken<T> tk{-1, 0, nullptr, nullptr, nullptr, nullptr, nullptr, 0};
  int seq_len = pos;
  if (g.token_pending) {
    const int phys = token_phys(g, ta.pt, b, pos);
    if (phys >= 0) {
      seq_len = pos + 1;
      tk = make_step_token<T>(g, ta.step, b, h, pos, phys, ta.k_new, ta.v_new, ta.kc, ta.vc, ta.A);
    }
  }
  const int n_pages = min((seq_len + g.P - 1) / g.P, g.max_pages);
  score_role<T, D, kScoreIters>(g, blockIdx.x * PPB, q + b * q_bstride + (int64_t)h * g.G * D,
                                dg + bh * g.max_pages * 2 * D, n_pages, scores + bh * g.max_pages,
                                sq, tk);
}

template <typename T, int D>
hipError_t score_t(const Geometry& g, int step, const void* q, int64_t qbs,
                   const retro_kv_cache& c, const void* k_new, const void* v_new, float* scores,
                   hipStream_t s) {
  constexpr int PPB = 4 * ScoreShape<T, D>::PPW * kScoreIters;
  dim3 grid((g.max_pages + PPB - 1) / PPB, g.hk, g.batch);
  const size_t lds = sizeof(float) * g.G * D;
  const TokenArgs ta{step, k_new, v_new, c.k_cache, c.v_cache, c.page_table, c.last_loaded};
  score_kernel<T, D><<<grid, 256, lds, s>>>(g, (const T*)q, qbs, (T*)c.digest, c.seq_lens, scores,
                                            ta);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_score(const Geometry& g, int step, const void* q_cur, int64_t q_batch_stride,
                        const retro_kv_cache& c, const void* k_new, const void* v_new,
                        float* scores, hipStream_t s) {
  if (g.dtype == RETRO_BF16)
    return g.D == 128 ? score_t<bf16_t, 128>(g, step, q_cur, q_batch_stride, c, k_new, v_new, scores, s)
                      : score_t<bf16_t, 64>(g, step, q_cur, q_batch_stride, c, k_new, v_new, scores, s);
  return g.D == 128 ? score_t<float, 128>(g, step, q_cur, q_batch_stride, c, k_new, v_new, scores, s)
                    : score_t<float, 64>(g, step, q_cur, q_batch_stride, c, k_new, v_new, scores, s);
}

}  // namespace retro
