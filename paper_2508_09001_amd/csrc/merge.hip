// Combine of the attention splits and MergeOutput + CacheOutput (Alg. 1) with
// the normaliser-weighted merge of eq. (merged_attn_general):
//   merge((O_a, Z_a), (O_b, Z_b)) = ((e^Za O_a + e^Zb O_b) / (e^Za + e^Zb),
//                                    ln(e^Za + e^Zb)),
// evaluated relative to max(Z_a, Z_b); a side with Z = -inf contributes nothing.
// The same merge combines the per-split partial outputs of one row.
//
// Output cache ring: row tau lives in slot tau mod W.  One workgroup per
// (sequence, query head, row) updates its own slot; rows 0 and W share a slot
// ((t-W) mod W == t mod W), so one workgroup handles both, reading the slot for
// row 0 before row W overwrites it.
#include "internal.h"

namespace retro {
namespace {

struct MergeArgs {
  Geometry g;
  int step;
  int mode;  // 0: splits -> part; 1: part -> cache; 2: splits -> cache
  const float* o_ws;
  const float* l_ws;
  const int32_t* nsel;
  const float* o_part;
  const float* l_part;
  float* o_part_out;
  float* l_part_out;
  float* o_cache;
  float* l_cache;
  float* o_out;
  float* l_out;
};

template <int D>
struct Row {
  static constexpr int E = D / 64;  // elements per thread
  float o[E];
  float z;
};

// The partial (O, Z) of row r for this workgroup's query head.
template <int D>
__device__ Row<D> partial(const MergeArgs& a, int b, int qh, int r) {
  const Geometry& g = a.g;
  Row<D> res;
  const int e0 = threadIdx.x * Row<D>::E;
  if (a.mode == 1) {
    const int64_t idx = ((int64_t)b * (g.W + 1) + r) * g.hq + qh;
#pragma unroll
    for (int e = 0; e < Row<D>::E; ++e) res.o[e] = a.o_part[idx * D + e0 + e];
    res.z = a.l_part[idx];
    return res;
  }
  const int h = qh / g.G, gq = qh - h * g.G;
  const int bh = b * g.hk + h;
  const int rho = r * g.G + gq;
  const int nvs = (a.nsel[bh] + g.pages_per_split - 1) / g.pages_per_split;
  const int64_t base = (int64_t)bh * g.n_splits * g.R + rho;
  float zmax = -INFINITY;
  for (int s = 0; s < nvs; ++s) zmax = fmaxf(zmax, a.l_ws[base + (int64_t)s * g.R]);
#pragma unroll
  for (int e = 0; e < Row<D>::E; ++e) res.o[e] = 0.f;
  if (zmax == -INFINITY) {
    res.z = -INFINITY;
    return res;
  }
  float wsum = 0.f;
  for (int s = 0; s < nvs; ++s) {
    const int64_t ri = base + (int64_t)s * g.R;
    const float w = __expf(a.l_ws[ri] - zmax);
    wsum += w;
#pragma unroll
    for (int e = 0; e < Row<D>::E; ++e) res.o[e] += w * a.o_ws[ri * D + e0 + e];
  }
  const float inv = 1.f / wsum;
#pragma unroll
  for (int e = 0; e < Row<D>::E; ++e) res.o[e] *= inv;
  res.z = zmax + __logf(wsum);
  return res;
}

template <int D>
__device__ Row<D> lse_merge(const Row<D>& x, const Row<D>& y) {
  Row<D> r;
  const float m = fmaxf(x.z, y.z);
  if (m == -INFINITY) {
#pragma unroll
    for (int e = 0; e < Row<D>::E; ++e) r.o[e] = 0.f;
    r.z = -INFINITY;
    return r;
  }
  const float wa = __expf(x.z - m), wb = __expf(y.z - m);
  const float inv = 1.f / (wa + wb);
#pragma unroll
  for (int e = 0; e < Row<D>::E; ++e) r.o[e] = (wa * x.o[e] + wb * y.o[e]) * inv;
  r.z = m + __logf(wa + wb);
  return r;
}

template <int D>
__device__ void put(float* o, float* z, int64_t idx, const Row<D>& v) {
  const int e0 = threadIdx.x * Row<D>::E;
#pragma unroll
  for (int e = 0; e < Row<D>::E; ++e) o[idx * D + e0 + e] = v.o[e];
  if (threadIdx.x == 0) z[idx] = v.z;
}

template <int D>
__device__ Row<D> get(const float* o, const float* z, int64_t idx) {
  Row<D> v;
  const int e0 = threadIdx.x * Row<D>::E;
#pragma unroll
  for (int e = 0; e < Row<D>::E; ++e) v.o[e] = o[idx * D + e0 + e];
  v.z = z[idx];
  return v;
}

template <int D>
__global__ void __launch_bounds__(64) combine_merge_kernel(MergeArgs a) {
  const Geometry& g = a.g;
  const int W = g.W;
  const int x = blockIdx.x, qh = blockIdx.y, b = blockIdx.z;
  const int64_t out_row = (int64_t)b * (W + 1);  // first row index of this sequence

  if (a.mode == 0) {  // plain combine of the splits for row x
    const Row<D> v = partial<D>(a, b, qh, x);
    put<D>(a.o_part_out, a.l_part_out, (out_row + x) * g.hq + qh, v);
    return;
  }

  Row<D> zero;
#pragma unroll
  for (int e = 0; e < Row<D>::E; ++e) zero.o[e] = 0.f;
  zero.z = -INFINITY;

  // rows handled here: x in [1, W) -> row x; x == 0 -> rows 0 and W
  const int rows[2] = {x, W};
  const int nrows = (x == 0 && W > 0) ? 2 : 1;
  for (int k = 0; k < nrows; ++k) {
    const int r = rows[k];
    const int tau = a.step - W + r;
    const int64_t oi = (out_row + r) * g.hq + qh;
    if (tau < 0) {
      put<D>(a.o_out, a.l_out, oi, zero);
      continue;
    }
    const Row<D> part = partial<D>(a, b, qh, r);
    if (r == W) {
      put<D>(a.o_out, a.l_out, oi, part);
      if (W > 0) {
        __syncthreads();  // row 0 of this workgroup has read the shared slot
        put<D>(a.o_cache, a.l_cache, ((int64_t)b * W + (a.step % W)) * g.hq + qh, part);
      }
      continue;
    }
    const int64_t ci = ((int64_t)b * W + (tau % W)) * g.hq + qh;
    const Row<D> merged = lse_merge<D>(get<D>(a.o_cache, a.l_cache, ci), part);
    put<D>(a.o_out, a.l_out, oi, merged);
    if (r > 0) put<D>(a.o_cache, a.l_cache, ci, merged);
  }
}

}  // namespace

hipError_t launch_combine_merge(const Geometry& g, int step, int mode, const float* o_ws,
                                const float* l_ws, const int32_t* num_selected,
                                const float* o_part, const float* l_part, float* o_part_out,
                                float* l_part_out, const retro_output_cache* oc, float* o_out,
                                float* lse_out, hipStream_t s) {
  MergeArgs a;
  a.g = g;
  a.step = step;
  a.mode = mode;
  a.o_ws = o_ws;
  a.l_ws = l_ws;
  a.nsel = num_selected;
  a.o_part = o_part;
  a.l_part = l_part;
  a.o_part_out = o_part_out;
  a.l_part_out = l_part_out;
  a.o_cache = oc ? oc->o_cache : nullptr;
  a.l_cache = oc ? oc->lse_cache : nullptr;
  a.o_out = o_out;
  a.l_out = lse_out;
  const int gx = (mode == 0) ? g.W + 1 : (g.W > 0 ? g.W : 1);
  dim3 grid(gx, g.hq, g.batch);
  if (g.D == 128)
    combine_merge_kernel<128><<<grid, 64, 0, s>>>(a);
  else
    combine_merge_kernel<64><<<grid, 64, 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace retro
