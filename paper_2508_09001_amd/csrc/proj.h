// Projections of the multi-layer decode (proj.hip), as the C entry points in
// api.hip use them.
#pragma once

#include "internal.h"

namespace retro {
// The query / key / value projections of a decoder layer's window rows with
// UpdateKV of the n_upd past rows folded in (proj.hip); bf16 only.
hipError_t launch_project_qkv_update(const Geometry& g, const retro_kv_cache& c, const void* x,
                                     int k, const void* w_packed, int n_upd, void* q,
                                     void* k_new, void* v_new, hipStream_t s);
bool project_qkv_update_supported(const Geometry& g, int k);

}  // namespace retro
