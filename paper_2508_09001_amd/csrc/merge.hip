// Combine of the attention splits and MergeOutput + CacheOutput (Alg. 1) with
// the normaliser-weighted merge of eq. (merged_attn_general):
//   merge((O_a, Z_a), (O_b, Z_b)) = ((e^Za O_a + e^Zb O_b) / (e^Za + e^Zb),
//                                    ln(e^Za + e^Zb)),
// evaluated relative to max(Z_a, Z_b); a side with Z = -inf contributes nothing.
// The same merge combines the per-split partial outputs of one row.
//
// One wavefront per (sequence, query head, row slot); lane l owns elements
// [l*E, l*E+E) of the d outputs.  Split normalisers are read one per lane and
// reduced across the wavefront; split outputs and the cache slot are all
// requested before any is used.
//
// Output cache ring: row tau lives in slot tau mod W.  Slot x of a wavefront:
// x in [1, W) -> row x; x == 0 -> rows 0 and W, which share a slot
// ((t-W) mod W == t mod W): the slot is read for row 0 before row W overwrites
// it, in program order of the same lanes.
#include "internal.h"

namespace retro {
namespace {

constexpr int kWaves = 4;  // wavefronts (work units) per workgroup

struct MergeArgs {
  Geometry g;
  int step;
  int mode;  // 0: splits -> part; 1: part -> cache; 2: splits -> cache
  int xs;    // row slots per query head
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
  static constexpr int E = D / 64;
  float o[E];
  float z;
};

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x = fmaxf(x, __shfl_xor(x, m));
  return x;
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m);
  return x;
}

// Combine the splits of row rho of (b, h): sum_s e^{Z_s} O_s / sum_s e^{Z_s}.
template <int D>
__device__ Row<D> combine_splits(const MergeArgs& a, int bh, int rho) {
  const Geometry& g = a.g;
  const int lane = threadIdx.x & 63;
  const int e0 = lane * Row<D>::E;
  const int nvs = min((a.nsel[bh] + g.pages_per_split - 1) / g.pages_per_split, g.n_splits);
  const int64_t base = (int64_t)bh * g.n_splits * g.R + rho;
  Row<D> res;
#pragma unroll
  for (int e = 0; e < Row<D>::E; ++e) res.o[e] = 0.f;
  float zmax = -INFINITY;
  for (int s0 = 0; s0 < nvs; s0 += 64) {
    const float z = (s0 + lane < nvs) ? a.l_ws[base + (int64_t)(s0 + lane) * g.R] : -INFINITY;
    zmax = fmaxf(zmax, z);
  }
  zmax = wave_max(zmax);
  if (zmax == -INFINITY) {
    res.z = -INFINITY;
    return res;
  }
  float wsum = 0.f;
  for (int s0 = 0; s0 < nvs; s0 += 64) {
    const int s = s0 + lane;
    const float w = (s < nvs) ? __expf(a.l_ws[base + (int64_t)s * g.R] - zmax) : 0.f;
    wsum += w;
    const int cnt = min(64, nvs - s0);
    // 8 split rows in flight at a time
    for (int j0 = 0; j0 < cnt; j0 += 8) {
      float v[8][Row<D>::E];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int ss = s0 + min(j0 + j, cnt - 1);
#pragma unroll
        for (int e = 0; e < Row<D>::E; ++e)
          v[j][e] = a.o_ws[(base + (int64_t)ss * g.R) * D + e0 + e];
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float wj = __shfl(w, j0 + j);
        if (j0 + j < cnt) {
#pragma unroll
          for (int e = 0; e < Row<D>::E; ++e) res.o[e] += wj * v[j][e];
        }
      }
    }
  }
  wsum = wave_sum(wsum);
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
  const int e0 = (threadIdx.x & 63) * Row<D>::E;
#pragma unroll
  for (int e = 0; e < Row<D>::E; ++e) o[idx * D + e0 + e] = v.o[e];
  if ((threadIdx.x & 63) == 0) z[idx] = v.z;
}

template <int D>
__device__ Row<D> get(const float* o, const float* z, int64_t idx) {
  Row<D> v;
  const int e0 = (threadIdx.x & 63) * Row<D>::E;
#pragma unroll
  for (int e = 0; e < Row<D>::E; ++e) v.o[e] = o[idx * D + e0 + e];
  v.z = z[idx];
  return v;
}

template <int D>
__device__ Row<D> partial(const MergeArgs& a, int b, int h, int gq, int r) {
  const Geometry& g = a.g;
  if (a.mode == 1) return get<D>(a.o_part, a.l_part, ((int64_t)b * (g.W + 1) + r) * g.hq + h * g.G + gq);
  return combine_splits<D>(a, b * g.hk + h, r * g.G + gq);
}

template <int D>
__global__ void __launch_bounds__(64 * kWaves) combine_merge_kernel(MergeArgs a) {
  const Geometry& g = a.g;
  const int W = g.W;
  // units ordered (sequence, KV head, query head of the group, row slot), spread
  // so that a KV head's units share the XCD its attention splits ran on
  const int nunits = g.batch * g.hq * a.xs;
  int u = xcd_remap(blockIdx.x, gridDim.x) * kWaves + (threadIdx.x >> 6);
  if (u >= nunits) return;  // uniform per wavefront; no barrier below
  const int x = u % a.xs;
  u /= a.xs;
  const int gq = u % g.G;
  u /= g.G;
  const int h = u % g.hk, b = u / g.hk;
  const int qh = h * g.G + gq;
  const int64_t out_row = (int64_t)b * (W + 1);

  if (a.mode == 0) {  // plain combine of the splits for row x
    put<D>(a.o_part_out, a.l_part_out, (out_row + x) * g.hq + qh, partial<D>(a, b, h, gq, x));
    return;
  }

  Row<D> zero;
#pragma unroll
  for (int e = 0; e < Row<D>::E; ++e) zero.o[e] = 0.f;
  zero.z = -INFINITY;

  const int r0 = x;
  const int tau0 = a.step - W + r0;
  if (r0 == W) {  // W == 0: the current row only
    put<D>(a.o_out, a.l_out, (out_row + r0) * g.hq + qh, partial<D>(a, b, h, gq, r0));
    return;
  }
  if (tau0 < 0) {
    put<D>(a.o_out, a.l_out, (out_row + r0) * g.hq + qh, zero);
  } else {
    const int64_t ci = ((int64_t)b * W + (tau0 % W)) * g.hq + qh;
    const Row<D> cached = get<D>(a.o_cache, a.l_cache, ci);
    const Row<D> merged = lse_merge<D>(cached, partial<D>(a, b, h, gq, r0));
    put<D>(a.o_out, a.l_out, (out_row + r0) * g.hq + qh, merged);
    if (r0 > 0) put<D>(a.o_cache, a.l_cache, ci, merged);
  }
  if (r0 == 0) {  // the current row: output, and push into slot t mod W
    const Row<D> cur = partial<D>(a, b, h, gq, W);
    put<D>(a.o_out, a.l_out, (out_row + W) * g.hq + qh, cur);
    put<D>(a.o_cache, a.l_cache, ((int64_t)b * W + (a.step % W)) * g.hq + qh, cur);
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
  a.xs = (mode == 0) ? g.W + 1 : (g.W > 0 ? g.W : 1);
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
  const int64_t units = (int64_t)g.batch * g.hq * a.xs;
  const unsigned blocks = (unsigned)((units + kWaves - 1) / kWaves);
  if (g.D == 128)
    combine_merge_kernel<128><<<blocks, 64 * kWaves, 0, s>>>(a);
  else
    combine_merge_kernel<64><<<blocks, 64 * kWaves, 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace retro
