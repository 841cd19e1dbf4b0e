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
#include "roles.h"

namespace retro {
namespace {

constexpr int kWaves = 2;  // wavefronts (work units) per workgroup: 256 workgroups at the headline shape, one per CU

__device__ __forceinline__ void update_last_loaded(const MergeArgs& a, int bh) {
  const Geometry& g = a.g;
  const int lane = threadIdx.x & 63;
  const int k = a.nsel[bh];
  const int tok = a.tok_upd[bh];
  const int32_t* srow = a.sel_upd + (int64_t)bh * g.k_max;
  int32_t* arow = a.a_upd + (int64_t)bh * g.max_pages;
  for (int i = lane; i < k && i < g.k_max; i += 64) {
    const int p = srow[i];
    if (p >= 0 && p < g.max_pages) arow[p] = a.step;
  }
  if (lane == 0 && tok >= 0 && tok < g.max_pages) arow[tok] = a.step - 1;
}

// GS: splits whose rows are loaded and folded in together, the smallest power
// of two (at most 32) covering the launch's splits
template <int D, int GS>
__global__ void __launch_bounds__(64 * kWaves) combine_merge_kernel(MergeArgs a) {
  // units ordered (sequence, KV head, query head of the group, row slot), spread
  // so that a KV head's units share the XCD its attention splits ran on
  const Geometry& g = a.g;
  const int nunits = g.batch * g.hq * a.xs;
  const int mblocks = (nunits + kWaves - 1) / kWaves;
  // A bounded wait of the launch that produced the partials ran out (or it
  // refused a workspace of another geometry): the partials and the selection
  // are not to be trusted, so the outputs are NaN and the caller's state (the
  // output cache, last_loaded, seq_lens) is left as it was.
  const bool failed = a.err && *a.err != 0;
  if ((int)blockIdx.x >= mblocks) {
    // workgroups past the merge units: Alg. 2's last_loaded update, one KV
    // head per wavefront
    const int bh = ((int)blockIdx.x - mblocks) * kWaves + (threadIdx.x >> 6);
    if (bh < g.batch * g.hk && !failed) update_last_loaded(a, bh);
    return;
  }
  // the wavefront index as a uniform value: the unit's indices and row offsets
  // then stay in scalar registers
  const int u = xcd_remap(blockIdx.x, mblocks) * kWaves + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (u >= nunits) return;  // uniform per wavefront; no barrier follows
  if (failed) {
    poison_unit<D>(a, unit_pos(a, u));
    return;
  }
  merge_unit<D, GS>(a, unit_pos(a, u));
  if (blockIdx.x == 0 && threadIdx.x < 64 && g.token_pending && a.seq_lens) {
    // after the unit's own loads (the two lookups here are dependent): the
    // first wavefront advances every sequence; no other workgroup of this
    // launch reads seq_lens
    for (int b = threadIdx.x; b < g.batch; b += 64) {
      const int pos = a.seq_lens[b];
      if (token_phys(g, a.pt, b, pos) >= 0) a.seq_lens[b] = pos + 1;
    }
  }
}

}  // namespace

MergeArgs make_merge_args(const Geometry& g, int step, int mode, const float* o_ws,
                          const float* l_ws, const int32_t* num_selected, const float* o_part,
                          const float* l_part, float* o_part_out, float* l_part_out,
                          const retro_output_cache* oc, float* o_out, float* lse_out) {
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
  a.seq_lens = nullptr;
  a.pt = nullptr;
  a.a_upd = nullptr;
  a.sel_upd = nullptr;
  a.tok_upd = nullptr;
  a.err = nullptr;
  return a;
}

hipError_t launch_combine_merge(const Geometry& g, int step, int mode, const float* o_ws,
                                const float* l_ws, const int32_t* num_selected,
                                const float* o_part, const float* l_part, float* o_part_out,
                                float* l_part_out, const retro_output_cache* oc, float* o_out,
                                float* lse_out, const retro_kv_cache* cache, hipStream_t s,
                                const int32_t* selected, const int32_t* tok_upd,
                                const int32_t* err) {
  MergeArgs a = make_merge_args(g, step, mode, o_ws, l_ws, num_selected, o_part, l_part,
                                o_part_out, l_part_out, oc, o_out, lse_out);
  if (cache) {
    a.seq_lens = cache->seq_lens;
    a.pt = cache->page_table;
  }
  a.err = err;
  int64_t upd_blocks = 0;
  if (selected && tok_upd) {
    if (!cache || !num_selected) return hipErrorInvalidValue;
    a.a_upd = cache->last_loaded;
    a.sel_upd = selected;
    a.tok_upd = tok_upd;
    upd_blocks = ((int64_t)g.batch * g.hk + kWaves - 1) / kWaves;
  }
  const int64_t units = (int64_t)g.batch * g.hq * a.xs;
  const unsigned blocks = (unsigned)((units + kWaves - 1) / kWaves + upd_blocks);
  const int ns = g.n_splits;
  if (g.D == 128) {
    if (ns <= 2) combine_merge_kernel<128, 2><<<blocks, 64 * kWaves, 0, s>>>(a);
    else if (ns <= 4) combine_merge_kernel<128, 4><<<blocks, 64 * kWaves, 0, s>>>(a);
    else if (ns <= 8) combine_merge_kernel<128, 8><<<blocks, 64 * kWaves, 0, s>>>(a);
    else if (ns <= 16) combine_merge_kernel<128, 16><<<blocks, 64 * kWaves, 0, s>>>(a);
    else combine_merge_kernel<128, 32><<<blocks, 64 * kWaves, 0, s>>>(a);
  } else {
    if (ns <= 2) combine_merge_kernel<64, 2><<<blocks, 64 * kWaves, 0, s>>>(a);
    else if (ns <= 4) combine_merge_kernel<64, 4><<<blocks, 64 * kWaves, 0, s>>>(a);
    else if (ns <= 8) combine_merge_kernel<64, 8><<<blocks, 64 * kWaves, 0, s>>>(a);
    else if (ns <= 16) combine_merge_kernel<64, 16><<<blocks, 64 * kWaves, 0, s>>>(a);
    else combine_merge_kernel<64, 32><<<blocks, 64 * kWaves, 0, s>>>(a);
  }
  return hipGetLastError();
}

}  // namespace retro
