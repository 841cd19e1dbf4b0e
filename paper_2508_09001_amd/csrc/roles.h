// Device-side building blocks ("roles") of the decode step, shared by the
// one-phase kernels behind the separate entry points and by the fused step
// kernel.  Every role uses all threads of its workgroup (any multiple of 64
// threads unless stated) and takes its LDS from the caller.
#pragma once

#include <type_traits>

#include "internal.h"

namespace retro {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kMaxPieces = 4;       // 16-byte staging registers per thread per chunk (attention kernel)
constexpr int kMaxSplitPages = 64;  // selected pages per attention split

// Device-coherent accesses (sc1: written through / read past the per-XCD L2s)
// for data handed between workgroups of one launch without fences.  Vector
// forms go through a buffer resource over [base, base + 2 GiB) (byte offsets;
// the host keeps such buffers below that size).
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4v __attribute__((ext_vector_type(4)));
constexpr int kCpolSc1 = 16;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t coherent_rsrc(const void* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, 0x7fffffff, 0x00020000);
}
template <bool COH, typename V>
__device__ __forceinline__ void put_c(V* p, V v) {
  if constexpr (COH) __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  else *p = v;
}
template <bool COH, typename V>
__device__ __forceinline__ V get_c(const V* p) {
  if constexpr (COH) return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  else return *p;
}

// A load through the scalar data cache (constant address space) from an
// address that is the same for the whole wavefront.  Its completion is counted
// apart from the vector loads', so waiting for it does not wait for the vector
// loads issued before it.  Only for memory that no workgroup of the launch
// writes before the read: the scalar cache is not kept coherent within a
// launch (it starts empty at every launch).
template <typename V>
__device__ __forceinline__ V sload(const V* p) {
  return *(const __attribute__((address_space(4))) V*)p;
}

// The thread's index in the workgroup, as a value the compiler cannot move:
// values computed from the index alone would otherwise be hoisted and kept
// live (in registers the later phases of a kernel then lack) across phases.
__device__ __forceinline__ int thread_index() {
  int t = threadIdx.x;
  asm volatile("" : "+v"(t));
  return t;
}

// Order-preserving map of a float to 32 bits: larger float -> larger key; -0 == +0.
__device__ __forceinline__ uint32_t order_key(float s) {
  uint32_t u = __float_as_uint(s);
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// ---- cross-lane moves without the LDS crossbar (DPP, gfx950 permlane swaps)
template <int CTRL, int ROW_MASK = 0xF, bool BOUND_ZERO = true>
__device__ __forceinline__ int dpp_i(int x) {
  return __builtin_amdgcn_update_dpp(0, x, CTRL, ROW_MASK, 0xF, BOUND_ZERO);
}
template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, true));
}
constexpr int kDppXor1 = 0xB1;       // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;       // quad_perm [2,3,0,1]
constexpr int kDppShl4 = 0x104;      // lane i reads lane i+4 of its 16-lane row
constexpr int kDppShl8 = 0x108;
constexpr int kDppHalfMirror = 0x141;
constexpr int kDppMirror = 0x140;

// Values of the other 16-lane rows at the same column: {even row, odd row} of
// each row pair, then {rows 0-1, rows 2-3}.
__device__ __forceinline__ float rows_pair_max(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
}
__device__ __forceinline__ float rows_half_max(float x) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
}
__device__ __forceinline__ float rows_pair_sum(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(a[0]) + __uint_as_float(a[1]);
}
__device__ __forceinline__ float rows_half_sum(float x) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(a[0]) + __uint_as_float(a[1]);
}
// max / sum of one column over the four 16-lane rows, in every lane
__device__ __forceinline__ float col_max4(float x) { return rows_half_max(rows_pair_max(x)); }
__device__ __forceinline__ float col_sum4(float x) { return rows_half_sum(rows_pair_sum(x)); }

// max / sum over the whole wavefront, in every lane
__device__ __forceinline__ float wave_max(float x) {
  x = fmaxf(x, dpp_f<kDppXor1>(x));
  x = fmaxf(x, dpp_f<kDppXor2>(x));
  x = fmaxf(x, dpp_f<kDppHalfMirror>(x));
  x = fmaxf(x, dpp_f<kDppMirror>(x));
  return col_max4(x);
}
__device__ __forceinline__ float wave_sum(float x) {
  x = x + dpp_f<kDppXor1>(x);
  x = x + dpp_f<kDppXor2>(x);
  x = x + dpp_f<kDppHalfMirror>(x);
  x = x + dpp_f<kDppMirror>(x);
  return col_sum4(x);
}
__device__ __forceinline__ uint32_t wave_umin(uint32_t x) {
  x = min(x, (uint32_t)dpp_i<kDppXor1, 0xF, false>((int)x));
  x = min(x, (uint32_t)dpp_i<kDppXor2, 0xF, false>((int)x));
  x = min(x, (uint32_t)dpp_i<kDppHalfMirror, 0xF, false>((int)x));
  x = min(x, (uint32_t)dpp_i<kDppMirror, 0xF, false>((int)x));
  auto a = __builtin_amdgcn_permlane16_swap(x, x, false, false);
  x = min((uint32_t)a[0], (uint32_t)a[1]);
  auto b = __builtin_amdgcn_permlane32_swap(x, x, false, false);
  return min((uint32_t)b[0], (uint32_t)b[1]);
}
__device__ __forceinline__ uint32_t wave_umax(uint32_t x) {
  x = max(x, (uint32_t)dpp_i<kDppXor1, 0xF, false>((int)x));
  x = max(x, (uint32_t)dpp_i<kDppXor2, 0xF, false>((int)x));
  x = max(x, (uint32_t)dpp_i<kDppHalfMirror, 0xF, false>((int)x));
  x = max(x, (uint32_t)dpp_i<kDppMirror, 0xF, false>((int)x));
  auto a = __builtin_amdgcn_permlane16_swap(x, x, false, false);
  x = max((uint32_t)a[0], (uint32_t)a[1]);
  auto b = __builtin_amdgcn_permlane32_swap(x, x, false, false);
  return max((uint32_t)b[0], (uint32_t)b[1]);
}

// Inclusive prefix sum over a wavefront: within 16-lane rows (shift right by
// 1, 2, 4, 8; missing lanes read 0), then across rows (row broadcasts).
__device__ __forceinline__ int wave_inclusive_scan(int x) {
  x += dpp_i<0x111>(x);
  x += dpp_i<0x112>(x);
  x += dpp_i<0x114>(x);
  x += dpp_i<0x118>(x);
  x += dpp_i<0x142, 0xA, false>(x);  // rows 1, 3 add the last lane of rows 0, 2
  x += dpp_i<0x143, 0xC, false>(x);  // rows 2, 3 add lane 31
  return x;
}

// Exclusive prefix sum over the workgroup (at most 16 wavefronts); sh >= 16 ints.
__device__ __forceinline__ int block_exclusive_scan(int v, int* sh) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const int x = wave_inclusive_scan(v);
  if (lane == 63) sh[wave] = x;
  __syncthreads();
  int off = 0;
  for (int w = 0; w < nw; ++w)
    if (w < wave) off += sh[w];
  __syncthreads();
  return off + x - v;
}

// ============================================================================
// Score role: eq. (quest_score) for a block of consecutive logical pages of one
// (sequence, KV head), in the fixed fp32 order (products rounded, pairwise sum
// over the d terms in index order, head sums in order, + 0.0f).  A page's digest
// row is read as 16-byte vectors by LPP = d / VEC consecutive lanes, lane c
// holding elements [c*VEC, (c+1)*VEC): the first log2(VEC) tree levels are
// in-lane, the rest pair neighbouring lanes (xor 1, 2, ...).
// ============================================================================
template <typename T, int D>
struct ScoreShape {
  static constexpr int LPP = 16;                    // lanes per page: one DPP row
  static constexpr int VEC = D / LPP;               // digest elements per lane
  static constexpr int WORDS = VEC * sizeof(T) / 4; // 32-bit words per lane per digest half
  static constexpr int PPW = 64 / LPP;              // pages per wavefront and pass
};

template <int WORDS>
__device__ __forceinline__ void load_words(const void* p, uint32_t* w) {
  if constexpr (WORDS == 2) {
    const uint2 u = *reinterpret_cast<const uint2*>(p);
    w[0] = u.x;
    w[1] = u.y;
  } else {
#pragma unroll
    for (int i = 0; i < WORDS; i += 4) {
      const uint4 u = reinterpret_cast<const uint4*>(p)[i / 4];
      w[i] = u.x;
      w[i + 1] = u.y;
      w[i + 2] = u.z;
      w[i + 3] = u.w;
    }
  }
}

template <int WORDS>
__device__ __forceinline__ void store_words(void* p, const uint32_t* w) {
  if constexpr (WORDS == 2) {
    *reinterpret_cast<uint2*>(p) = make_uint2(w[0], w[1]);
  } else {
#pragma unroll
    for (int i = 0; i < WORDS; i += 4)
      reinterpret_cast<uint4*>(p)[i / 4] = make_uint4(w[i], w[i + 1], w[i + 2], w[i + 3]);
  }
}

template <typename T, int WORDS>
__device__ __forceinline__ void words_to_f32(const uint32_t* w, float* out) {
  if constexpr (sizeof(T) == 2) {
#pragma unroll
    for (int i = 0; i < WORDS; ++i) {
      out[2 * i] = __uint_as_float(w[i] << 16);
      out[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
  } else {
#pragma unroll
    for (int i = 0; i < WORDS; ++i) out[i] = __uint_as_float(w[i]);
  }
}

// inverse of words_to_f32 for values exactly representable in T
template <typename T, int WORDS>
__device__ __forceinline__ void f32_to_words(const float* in, uint32_t* w) {
  if constexpr (sizeof(T) == 2) {
#pragma unroll
    for (int i = 0; i < WORDS; ++i)
      w[i] = (__float_as_uint(in[2 * i]) >> 16) | (__float_as_uint(in[2 * i + 1]) & 0xFFFF0000u);
  } else {
#pragma unroll
    for (int i = 0; i < WORDS; ++i) w[i] = __float_as_uint(in[i]);
  }
}

// The step's own token, appended by the score block whose pages include it:
// AppendKV and the digest update.  Alg. 2's current-page rule (last_loaded of the
// token's page = step - 1) is applied by the selection (topk_role), which owns
// every last_loaded write of the step.
template <typename T>
struct StepToken {
  int lp;            // logical page of the token (-1: none)
  int slot;          // slot in the page
  const T* k;        // [d] key of this KV head
  const T* v;        // [d] value of this KV head
  T* k_row;          // the slot's key row (token-major page)
  T* v_col;          // the slot's value column (d-major page): element i at v_col[i * P]
};

// Physical page that receives the token at position pos of sequence b, or -1
// when its logical page is out of range or unmapped (the token is then skipped).
__device__ __forceinline__ int token_phys(const Geometry& g, const int32_t* pt, int b, int pos) {
  const int lp = pos / g.P;
  if (pos < 0 || lp >= g.max_pages) return -1;
  const int phys = pt[(int64_t)b * g.max_pages + lp];
  return (phys >= 0 && phys < g.num_phys) ? phys : -1;
}

// Length of sequence b during the step: seq_lens[b], plus the step's token
// when it is still pending (see Geometry::token_pending) and will be stored.
__device__ __forceinline__ int live_seq_len(const Geometry& g, const int32_t* seq_lens,
                                            const int32_t* pt, int b) {
  const int pos = seq_lens[b];
  return (g.token_pending && token_phys(g, pt, b, pos) >= 0) ? pos + 1 : pos;
}

// The token of KV head h of sequence b at position pos, stored in physical page
// phys (>= 0), as the score role appends it.
template <typename T>
__device__ __forceinline__ StepToken<T> make_step_token(const Geometry& g, int b, int h, int pos,
                                                        int phys, const void* k_new,
                                                        const void* v_new, void* kc, void* vc) {
  const int lp = pos / g.P, slot = pos - lp * g.P;
  const int64_t bh = (int64_t)b * g.hk + h;
  const int64_t ph = (int64_t)phys * g.hk + h;
  StepToken<T> tk;
  tk.lp = lp;
  tk.slot = slot;
  tk.k = reinterpret_cast<const T*>(k_new) + bh * g.D;
  tk.v = reinterpret_cast<const T*>(v_new) + bh * g.D;
  tk.k_row = reinterpret_cast<T*>(kc) + (ph * g.P + slot) * g.D;
  tk.v_col = reinterpret_cast<T*>(vc) + ph * g.D * g.P + slot;
  return tk;
}

// Scores pages [page0, page0 + blockDim/64 * PPW * ITERS) of one (sequence, KV
// head).  A page is handled by one 16-lane row, lane c holding elements
// [c*VEC, (c+1)*VEC): the first log2(VEC) levels of the pairwise tree are
// in-lane, the last four pair lane c with c+1, c+2, c+4, c+8 through DPP (the
// left operand is always the lower index).  tok.lp < 0: no token to append.
// The workgroup scores pages [page0, page_end) (at most ITERS passes of four
// pages per wavefront; pass it covers the workgroup's pages it*nw*4 onwards).
// DEFER: the role stores nothing to global memory itself: the widened digest
// row of the token's page goes to dig_lds (2 * D elements of LDS: minimum,
// then maximum) and the token's key and value are left to the caller (the
// caller then issues every store of the phase from one wavefront, so that the
// others carry no pending store into the loads that follow).  Otherwise the
// row, the key and the value are stored here.  GC > 0: the group size is GC (== g.G), so
// the loop over the group's heads unrolls and the heads' reduction chains
// interleave (0.2 us per step at G = 4); 0: any g.G.
// The token and the number of pages of the sequence come from `tok_of(n_pages)`
// (returns the StepToken, sets n_pages), called once the digest and query loads
// are issued: its own loads (sequence length, page table) then overlap them.
// sq: 2 * G * D floats of LDS, where the group's queries are staged as
// max(q, 0) (first G * D) and min(q, 0) (the rest).
// `pre_barrier()` runs in every thread just before the barrier that publishes
// the staged queries to the workgroup; `publish(page, score)` hands each score
// of a page below n_pages on (called by one lane per page).  NT > 0: the
// workgroup has NT threads (else blockDim.x).  The digest loads depend on
// page0, page_end and drow only, and are not branched around (pages past the
// share read its last row, and their scores are not published), so they can
// go out before any other kernel argument has arrived.
template <typename T, int D, int ITERS, bool DEFER, int GC = 0, int NT = 0, typename TokOf,
          typename PreBarrier, typename Publish>
__device__ __forceinline__ void score_role(const Geometry& g, int page0, int page_end, const T* q,
                                           T* drow, float* sq, TokOf&& tok_of,
                                           PreBarrier&& pre_barrier, Publish&& publish,
                                           T* dig_lds = nullptr) {
#pragma clang fp contract(off)
  using S = ScoreShape<T, D>;
  const int tid = thread_index();
  const int nthreads = NT > 0 ? NT : (int)blockDim.x;
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6), nw = nthreads >> 6;
  const int c = lane % S::LPP;
  // every load before any wait: the group's queries (first: they are staged
  // before the barrier, and loads complete in order), digest rows (in bounds
  // of the [max_pages] row whatever the sequence length), the token's key.
  // Queries as 16-byte pieces, QR per thread (G * d <= 16 d elements), all
  // requested before any is converted, without a branch (threads past the
  // group's queries load its last piece and store nothing)
  constexpr int QV = 16 / sizeof(T);
  constexpr int QR = NT > 0 ? (16 * D + NT * QV - 1) / (NT * QV) : 2;
  const int gd = (GC > 0 ? GC : g.G) * D;
  uint4 qraw[QR];
#pragma unroll
  for (int r = 0; r < QR; ++r) {
    const int e = (tid + r * nthreads) * QV;
    qraw[r] = *reinterpret_cast<const uint4*>(q + min(e, gd - QV));
  }
  uint32_t raw[ITERS][2][S::WORDS];
  const int last_row = max(page_end - 1, 0);
#pragma unroll
  for (int it = 0; it < ITERS; ++it) {
    const int page = min(page0 + (it * nw + wave) * S::PPW + lane / S::LPP, last_row);
    const T* row = drow + (int64_t)page * 2 * D + c * S::VEC;
    load_words<S::WORDS>(row, raw[it][0]);
    load_words<S::WORDS>(row + D, raw[it][1]);
  }
  int n_pages = 0;
  const StepToken<T> tok = tok_of(n_pages);
  const bool has_tok = tok.lp >= 0 && tok.lp >= page0 && tok.lp < page_end;
  // the token's key and value, element tid, for the append at the end: read
  // now so that the append does not wait for a round trip of its own (every
  // workgroup running this role has at least 256 threads)
  static_assert(D <= 256, "one element per thread");
  T tok_k = T{}, tok_v = T{};
  if (!DEFER && has_tok) {  // uniform
    tok_k = tok.k[min(tid, D - 1)];
    tok_v = tok.v[min(tid, D - 1)];
  }
  // (converted where the token's page is scored, after the barrier)
  uint32_t kw[S::WORDS] = {};
  if (has_tok) load_words<S::WORDS>(tok.k + c * S::VEC, kw);
#pragma unroll
  for (int r = 0; r < QR; ++r) {
    const int e = (tid + r * nthreads) * QV;
    if (e < gd) {
      const uint32_t w[4] = {qraw[r].x, qraw[r].y, qraw[r].z, qraw[r].w};
      float f[QV];
      words_to_f32<T, 4>(w, f);
#pragma unroll
      for (int i = 0; i < QV; i += 4) {
        *reinterpret_cast<float4*>(sq + e + i) =
            make_float4(fmaxf(f[i], 0.f), fmaxf(f[i + 1], 0.f), fmaxf(f[i + 2], 0.f), fmaxf(f[i + 3], 0.f));
        *reinterpret_cast<float4*>(sq + gd + e + i) =
            make_float4(fminf(f[i], 0.f), fminf(f[i + 1], 0.f), fminf(f[i + 2], 0.f), fminf(f[i + 3], 0.f));
      }
    }
  }
  pre_barrier();
  __syncthreads();

  float score[ITERS];
#pragma unroll
  for (int it = 0; it < ITERS; ++it) {
    score[it] = 0.f;
    const int wpage0 = page0 + (it * nw + wave) * S::PPW;
    if (it > 0 && wpage0 >= page_end) break;  // uniform: no page of this pass
    const int page = wpage0 + lane / S::LPP;
    float lo[S::VEC], hi[S::VEC];
    words_to_f32<T, S::WORDS>(raw[it][0], lo);
    words_to_f32<T, S::WORDS>(raw[it][1], hi);
    if (has_tok && page == tok.lp) {  // widen (or start) the digest with the new key
      float kv[S::VEC];
      words_to_f32<T, S::WORDS>(kw, kv);
#pragma unroll
      for (int v = 0; v < S::VEC; ++v) {
        if (tok.slot == 0) {
          lo[v] = kv[v];
          hi[v] = kv[v];
        } else {
          if (kv[v] < lo[v]) lo[v] = kv[v];
          if (hi[v] < kv[v]) hi[v] = kv[v];
        }
      }
      T* row = (DEFER ? dig_lds : drow + (int64_t)page * 2 * D) + c * S::VEC;
      uint32_t w[S::WORDS];
      f32_to_words<T, S::WORDS>(lo, w);
      store_words<S::WORDS>(row, w);
      f32_to_words<T, S::WORDS>(hi, w);
      store_words<S::WORDS>(row + D, w);
    }
    float Ssum = 0.f;
    // head gq's sum over d (a perfect binary tree: in-lane, then across the
    // row's lanes), added to the running sum in head order
    auto head = [&](int gq) {
      float t[S::VEC];
#pragma unroll
      for (int v = 0; v < S::VEC; ++v) {
        // max(q*lo, q*hi) is the product with hi for q >= 0 and with lo for
        // q < 0 (lo <= hi, and rounding is monotone).  With q+ = max(q, 0)
        // and q- = min(q, 0) staged apart, that is fma(q-, lo, q+ * hi): one
        // of the two products is a zero, so the fma rounds the other one once,
        // as the plain product does.  Only a zero term's sign can differ,
        // which changes no sum with a nonzero term and is cleared by the
        // final + 0.0f otherwise, so the score is the same bit for bit.
        const float qp = sq[gq * D + c * S::VEC + v];
        const float qn = sq[gd + gq * D + c * S::VEC + v];
        t[v] = __builtin_fmaf(qn, lo[v], qp * hi[v]);
      }
#pragma unroll
      for (int w = 1; w < S::VEC; w *= 2)
#pragma unroll
        for (int i = 0; i + w < S::VEC; i += 2 * w) t[i] = t[i] + t[i + w];
      float s = t[0];
      s = s + dpp_f<kDppXor1>(s);
      s = s + dpp_f<kDppXor2>(s);
      s = s + dpp_f<kDppShl4>(s);
      s = s + dpp_f<kDppShl8>(s);
      Ssum = (gq == 0) ? s : Ssum + s;
    };
    if constexpr (GC > 0) {
#pragma unroll
      for (int gq = 0; gq < GC; ++gq) head(gq);
    } else {
      for (int gq = 0; gq < g.G; ++gq) head(gq);
    }
    score[it] = Ssum + 0.0f;
  }
  if (!DEFER && has_tok && tid < D) {
    tok.k_row[tid] = tok_k;
    tok.v_col[(int64_t)tid * g.P] = tok_v;
  }
#pragma unroll
  for (int it = 0; it < ITERS; ++it) {
    const int page = page0 + (it * nw + wave) * S::PPW + lane / S::LPP;
    if (page < n_pages && page < page_end && c == 0) publish(page, score[it]);
  }
}

// Pages of the step's budget for a sequence of `len` tokens: B / P with a fixed
// budget; with a relative one (the ablation of Sec. 4, Table 1's setting) the
// budget is max(B, floor(len * permille / 1000)) tokens, len counting the
// step's token.
__device__ __forceinline__ int budget_pages(const Geometry& g, int len) {
  int b = g.budget;
  if (g.budget_permille > 0) b = max(b, (int)((int64_t)len * g.budget_permille / 1000));
  return b / g.P;
}

// ============================================================================
// Top-k + mask role: PageSelect and UpdateAndBuildMask (Alg. 1, Alg. 2) for
// one (sequence, KV head); see topk.hip for the algorithm.
// ============================================================================
struct TopkArgs {
  Geometry g;
  int step;
  const float* scores;
  const int32_t* pt;
  int32_t* A;
  int32_t* selected;
  int32_t* mask;
  int32_t* num_selected;
  int32_t* sel_phys;  // physical ids of the kept pages, or null
};

constexpr int kTopkBins = 2048;    // bins of an 11-bit digit
constexpr int kTopkPasses = 3;     // 11 + 11 + 10 bits cover a 32-bit key
constexpr int kTopkHistWords = kTopkPasses * kTopkBins;  // one histogram per pass
constexpr int kTopkSmall = 32 + 4 + 256;  // ints: min/max exchange, pass result, per-(stripe, wave) counts

__device__ __forceinline__ uint64_t wave_ballot(bool p) { return __builtin_amdgcn_ballot_w64(p); }
// number of set bits of m in lanes below this one
__device__ __forceinline__ int lanes_below(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
}

// The selection itself, without its outputs: returns k, the pages kept, and
// calls `on_page(pos, p, a_old, phys)` for every stripe slot of every thread
// (p: logical page, a_old: its last_loaded value as Alg. 2 reads it, phys: its
// page-table entry; pos: its rank among the kept pages in page order, or -1
// when it is not kept or past the sequence).
// THREADS = blockDim.x threads (at most MAXW wavefronts); page i of the
// sequence is held by thread i mod THREADS in stripe i / THREADS (coalesced
// loads).  ceil(max_pages / THREADS) <= PER.  tok_lp: logical page written by
// this step's token (-1: none), read after `len_of()` (which may set it):
// Alg. 2's current-page rule applies to it, so its last_loaded entry is taken as
// step - 1.  `len_of()` gives the sequence's length in tokens (with the step's
// token when it is stored), which fixes n = its pages and the budget; it is called once
// the loads are issued.  hist: kTopkHistWords
// uint32 of LDS; small: kTopkSmall ints of LDS.
// `wait()` is called after the page-table and last_loaded loads are issued and
// before the scores are read.
template <int PER, int MAXW, typename LenOf, typename Wait, typename OnPage>
__device__ __forceinline__ int topk_core(const TopkArgs& ta, int bh, LenOf&& len_of, const int& tok_lp,
                                         uint32_t* hist, int* small, Wait&& wait,
                                         OnPage&& on_page) {
  constexpr int NCH = (PER * MAXW + 63) / 64;  // 64-entry chunks of the count table
  static_assert(PER * MAXW <= kTopkSmall - 36 && MAXW <= 16 && PER <= 32, "top-k shape");
  const int THREADS = blockDim.x, NW = THREADS >> 6;
  const Geometry& g = ta.g;
  const int step = ta.step;
  const int tid = thread_index(), lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int b = bh / g.hk;
  const float* srow = ta.scores + (int64_t)bh * g.max_pages;
  const int32_t* a_row = ta.A + (int64_t)bh * g.max_pages;
  const int32_t* p_row = ta.pt + (int64_t)b * g.max_pages;
  int* red = small;        // [32]
  int* res = small + 32;   // [4]: T's digit, keys above its bin, keys in it
  int* cnt = small + 36;   // [PER * NW]

  // Loads are issued for every stripe slot before the number of pages is known
  // (an in-bounds index stands in for slots past the row; their values are
  // not used), so none waits for another.
  const int last = g.max_pages - 1;
  int32_t a_old[PER], phys[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int idx = min(j * THREADS + tid, last);
    a_old[j] = a_row[idx];
    phys[j] = p_row[idx];
  }
  for (int i = tid; i < kTopkHistWords; i += THREADS) hist[i] = 0u;
  wait();
  float sv[PER];  // device-coherent loads: the scores may come from other XCDs of this launch
#pragma unroll
  for (int j = 0; j < PER; ++j)
    sv[j] = __hip_atomic_load(srow + min(j * THREADS + tid, last), __ATOMIC_RELAXED,
                              __HIP_MEMORY_SCOPE_AGENT);
  const int len = len_of();
  const int n = min((len + g.P - 1) / g.P, g.max_pages);
  auto valid = [&](int j) { return j * THREADS + tid < n; };
#pragma unroll
  for (int j = 0; j < PER; ++j)
    if (j * THREADS + tid == tok_lp) a_old[j] = step - 1;
  uint32_t key[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) key[j] = valid(j) ? order_key(sv[j]) : 0u;

  // rel = key - kmin over the valid keys; T is searched among rel values.
  uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
#pragma unroll
  for (int j = 0; j < PER; ++j)
    if (valid(j)) {
      kmin = min(kmin, key[j]);
      kmax = max(kmax, key[j]);
    }
  kmin = wave_umin(kmin);
  kmax = wave_umax(kmax);
  if (lane == 0) {
    red[wave] = (int)kmin;
    red[16 + wave] = (int)kmax;
  }
  __syncthreads();  // also orders the histogram clearing before the first pass
  kmin = wave_umin(lane < NW ? (uint32_t)red[lane] : 0xFFFFFFFFu);
  kmax = wave_umax(lane < NW ? (uint32_t)red[16 + lane] : 0u);
  const uint32_t range = kmax - kmin;
  const int nbits = range ? 32 - __clz((int)range) : 1;
  const int k = min(min(budget_pages(g, len), n), g.k_max);

  // Radix select: pass p histograms the next digit of the keys that still match
  // T's prefix into its own histogram.  After a barrier, wavefront 0 alone
  // scans it (descending bins, lane l owning 32 of them) and publishes T's
  // digit, the keys above its bin and the keys in it; the other wavefronts
  // wait at the next barrier (a scan by every wavefront would share the four
  // SIMDs between sixteen copies of the same work).
  uint64_t prefix = 0u;  // digits of T's rel fixed so far, bits [lo, nbits)
  int lo = nbits;
  uint32_t need = (uint32_t)k;  // keys still to take among those matching the prefix
  if (k > 0 && k < n) {
    int pass = 0;
#pragma unroll 1
    for (int hi = nbits; hi > 0; hi = lo, ++pass) {
      lo = max(hi - 11, 0);
      uint32_t* h = hist + pass * kTopkBins;
      const uint32_t dmask = (1u << (hi - lo)) - 1u;
#pragma unroll
      for (int j = 0; j < PER; ++j) {
        const uint64_t rel = key[j] - kmin;
        if (valid(j) && (rel >> hi) == prefix) atomicAdd(&h[(rel >> lo) & dmask], 1u);
      }
      __syncthreads();
      if (wave == 0) {
        const int base = kTopkBins - 32 * (lane + 1);
        uint32_t gs[8];  // totals of this lane's eight 4-bin groups (ascending bins)
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const uint4 u = *reinterpret_cast<const uint4*>(h + base + 4 * i);
          gs[i] = u.x + u.y + u.z + u.w;
        }
        uint32_t own = 0u;
#pragma unroll
        for (int i = 0; i < 8; ++i) own += gs[i];
        const uint32_t incl = (uint32_t)wave_inclusive_scan((int)own);
        uint32_t acc = incl - own;  // keys in higher bins
        const bool hit = acc < need && need <= incl;
        // the group holding T's digit (highest group first), then the bin in it
        int fgrp = 0;
        uint32_t facc = 0u;
        bool found = false;
#pragma unroll
        for (int i = 7; i >= 0; --i) {
          const bool f = !found && acc + gs[i] >= need;
          fgrp = f ? i : fgrp;
          facc = f ? acc : facc;
          found = found || f;
          acc += gs[i];
        }
        const uint4 u = *reinterpret_cast<const uint4*>(h + base + 4 * fgrp);
        const uint32_t gv[4] = {u.x, u.y, u.z, u.w};
        int fb = 0;
        uint32_t fc = 0u, fa = 0u;
        found = false;
        acc = facc;
#pragma unroll
        for (int i = 3; i >= 0; --i) {
          const bool f = !found && acc + gv[i] >= need;
          fb = f ? base + 4 * fgrp + i : fb;
          fc = f ? gv[i] : fc;
          fa = f ? acc : fa;
          found = found || f;
          acc += gv[i];
        }
        if (hit) {  // exactly one lane: need lies in its range of the running total
          res[0] = fb;
          res[1] = (int)fa;
          res[2] = (int)fc;
        }
      }
      __syncthreads();
      const int bin = res[0];
      const uint32_t above = (uint32_t)res[1], inbin = (uint32_t)res[2];
      need -= above;
      prefix = (prefix << (hi - lo)) | (uint32_t)bin;
      if (inbin == need) break;  // T's whole bin is kept: its prefix suffices
      if (lo > 0 && inbin <= 64) {
        // T is one of its bin's few keys: list them (in the next pass's
        // histogram, still zero) and let wavefront 0 rank them exactly (lane i
        // holds candidate i and counts the larger and equal ones through LDS
        // broadcast reads) instead of histogramming further digits.
        uint32_t* cand = hist + (pass + 1) * kTopkBins;  // [0]: count, [1..]: rel values
#pragma unroll
        for (int j = 0; j < PER; ++j) {
          const uint64_t rel = key[j] - kmin;
          if (valid(j) && (rel >> lo) == prefix) cand[1 + atomicAdd(&cand[0], 1u)] = (uint32_t)rel;
        }
        __syncthreads();
        if (wave == 0) {
          const uint32_t v = lane < (int)inbin ? cand[1 + lane] : 0u;
          uint32_t gt = 0u, eq = 0u;
          for (int j2 = 0; j2 < (int)inbin; ++j2) {
            const uint32_t w = cand[1 + j2];
            gt += w > v ? 1u : 0u;
            eq += w == v ? 1u : 0u;
          }
          const bool is_t = lane < (int)inbin && gt < need && need <= gt + eq;
          if (lane == __builtin_ctzll(wave_ballot(is_t))) {
            res[0] = (int)v;   // T's whole rel
            res[1] = (int)gt;  // candidates above T
          }
        }
        __syncthreads();
        prefix = (uint32_t)res[0];
        need -= (uint32_t)res[1];  // keys equal to T still to take
        lo = 0;
        break;
      }
    }
  }

  // Compaction in page order.  A kept page's output slot is the number of kept
  // pages below it: pages above T's prefix all count, pages tying with it count
  // up to `need` (lower page indices first).  Per stripe, ballots give the
  // counts below a lane inside its wavefront; an exclusive scan over the
  // (stripe, wavefront) count table, in page order, gives the rest.
  const bool all = k >= n;
  const bool some = k > 0 && k < n;
  uint32_t gt_bits = 0u, eq_bits = 0u;  // per stripe: above T's prefix / tying with it
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const uint64_t km = (uint64_t)(key[j] - kmin) >> lo;
    const bool v = valid(j);
    const bool gt = v && (all || (some && km > prefix));
    const bool eq = v && some && km == prefix;
    gt_bits |= (gt ? 1u : 0u) << j;
    eq_bits |= (eq ? 1u : 0u) << j;
    const int cg = __popcll(wave_ballot(gt)), ce = __popcll(wave_ballot(eq));
    if (lane == 0) cnt[j * NW + wave] = cg | (ce << 16);
  }
  __syncthreads();
  int sc[NCH];  // exclusive scan of the count table, entry c * 64 + lane
  int carry = 0;
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const int e = c * 64 + lane;
    const int val = e < PER * NW ? cnt[e] : 0;
    const int incl = wave_inclusive_scan(val) + carry;
    sc[c] = incl - val;
    carry = __builtin_amdgcn_readlane(incl, 63);
  }
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int e = j * NW + wave;
    int below = 0;
#pragma unroll
    for (int c = 0; c < NCH; ++c)
      if (e / 64 == c) below = __builtin_amdgcn_readlane(sc[c], e % 64);
    const bool is_gt = (gt_bits >> j) & 1u;
    const bool is_eq = (eq_bits >> j) & 1u;
    const int gb = (below & 0xFFFF) + lanes_below(wave_ballot(is_gt));
    const int eb = (below >> 16) + lanes_below(wave_ballot(is_eq));
    int pos = -1;
    if (is_gt) pos = gb + min(eb, (int)need);
    if (is_eq && eb < (int)need) pos = gb + eb;
    // pos < k always holds for a kept page; the test guards the writes
    on_page(pos < k ? pos : -1, j * THREADS + tid, a_old[j], phys[j]);
  }
  return k;
}

// Selection of KV head bh with its outputs: the selected pages in page order,
// their mask values M (last_loaded before the step) and physical pages, -1
// past the k kept ones, the count, and last_loaded set to the step for the kept
// pages (step - 1 for the token's page when it is not kept).  Arguments as
// topk_core's.  COH: the selection is read by other workgroups of the same
// launch, so it is stored device-coherently.
template <int PER, int MAXW, bool COH, typename LenOf, typename Wait>
__device__ __forceinline__ void topk_role(const TopkArgs& ta, int bh, LenOf&& len_of, int tok_lp,
                                          uint32_t* hist, int* small, Wait&& wait) {
  const Geometry& g = ta.g;
  const int step = ta.step;
  int32_t* a_row = ta.A + (int64_t)bh * g.max_pages;
  int32_t* sel_row = ta.selected + (int64_t)bh * g.k_max;
  int32_t* m_row = ta.mask + (int64_t)bh * g.k_max;
  int32_t* ph_row = ta.sel_phys ? ta.sel_phys + (int64_t)bh * g.k_max : nullptr;
  const int k = topk_core<PER, MAXW>(
      ta, bh, len_of, tok_lp, hist, small, wait, [&](int pos, int p, int a_old, int phys) {
        if (pos >= 0) {
          put_c<COH>(sel_row + pos, p);
          put_c<COH>(m_row + pos, a_old);
          a_row[p] = step;
          if (ph_row) put_c<COH>(ph_row + pos, (phys >= 0 && phys < g.num_phys) ? phys : -1);
        } else if (p == tok_lp) {
          a_row[p] = step - 1;  // the token's page, not kept
        }
      });
  const int tid = thread_index(), THREADS = blockDim.x;
  for (int i = k + tid; i < g.k_max; i += THREADS) {
    put_c<COH>(sel_row + i, -1);
    put_c<COH>(m_row + i, -1);
    if (ph_row) put_c<COH>(ph_row + i, -1);
  }
  if (tid == 0) put_c<COH>(ta.num_selected + bh, k);
}


// ============================================================================
// Attention role (see attend.hip for the design).
// ============================================================================
template <typename T, int D>
struct Tiles {
  static constexpr int VEC = 16 / sizeof(T);          // elements per 16 bytes
  static constexpr int KROW = D + VEC;                // padded LDS key row (elements)
  static constexpr int VROW = 16 + (sizeof(T) == 2 ? 8 : 4);  // padded V^T row
  static constexpr int K_ELEMS = 32 * KROW;
  static constexpr int V_ELEMS = 2 * D * VROW;
  static constexpr int BUF_ELEMS = K_ELEMS + V_ELEMS;
  static constexpr int KPR = D / VEC;                 // 16-byte pieces per key row
  static constexpr int VPR = 16 / VEC;                // pieces per 16-token V^T row
  static constexpr int TPP = VEC;                     // tokens per V piece
  static constexpr int K_PIECES = 32 * KPR;
  static constexpr int PIECES = K_PIECES + 2 * D * VPR;
};

struct AttendArgs {
  Geometry g;
  int step;
  float scale_log2;
  const void* q;
  const void* kc;
  const void* vc;
  const int32_t* pt;
  const int32_t* seq_lens;
  const int32_t* sel;
  const int32_t* msk;
  const int32_t* nsel;
  const int32_t* sel_phys;  // physical ids of the selected pages, or null (page-table lookup)
  float* o_ws;
  float* l_ws;
  // 16 bytes that no kernel writes (a line of the workspace): loads of chunk
  // pieces with no stored data read here instead of branching around the load,
  // so they never bring a line of the KV cache into a cache early
  const void* dummy;
  // the step's token, [batch][h_k][d], when another workgroup of the same
  // launch stores it into the cache (see attend_role's tok_pos); else null
  const void* tok_k;
  const void* tok_v;
};

AttendArgs make_attend_args(const Geometry& g, int step, const void* q_window,
                            const retro_kv_cache& c, const retro_selection& sel,
                            const int32_t* sel_phys, float* o_ws, float* l_ws, const void* dummy);


// The attention pass of one (sequence, KV head, row group, split).  Row-tile
// state and the query operands are set up first; `wait()` is then called (the
// fused step waits there for the page selection), and only then is the page
// list read.  Uses `lds` (2 * Tiles<T, D>::BUF_ELEMS elements, 16-byte aligned)
// and three int arrays of kMaxSplitPages entries; MAXP bounds the 16-byte pieces
// of a chunk per thread (ceil(Tiles::PIECES / threads)); PAIR computes chunks
// two at a time (more registers).  `seq_len_of()` gives the
// sequence length in effect; it is called once the page-list loads are issued.
// COH: the selection comes from, and the partials go to, other workgroups of
// the same launch: device-coherent loads and stores.
// The split's page list comes from the selection rows in memory (COH: written
// by other workgroups of the same launch) when `list` is a SelectionRows, else
// `list(tid, first, lp, m, phys)` gives thread tid's slot of it (slot tid of
// the selection row from `first` on: logical page, mask value, physical page;
// left as passed in for tid >= pages_per_split) and returns the number of
// selected pages of the row.
// tok_pos >= 0: the position of the step's token, which another workgroup of
// the same launch is storing into the cache: its key row and value column are
// taken from a.tok_k / a.tok_v into LDS instead (so no gather has to wait for
// that store); the cache supplies the page's other tokens, stored by earlier
// launches.  s_tok: one int of LDS.
// With a PresetList the caller has filled the split's page list itself before
// `wait()` returns (after a barrier): s_phys / s_len / s_mask for every slot
// of the split (-1 / 0 / 0 past the kept pages), *s_tok (the slot of the
// token's page, -1 if not in the split), and gives the number of kept pages
// and, for the first d threads, the token's key and value elements.
// With COH and a PresetList whose lse_tag is set, each wavefront publishes
// its rows' log-normalisers itself once its partial-output stores are
// acknowledged: one 64-bit word per (row, split), the launch's epoch (bit 31:
// *bad, the workgroup failed) over the value's bits, at lse_tag[(b * h_k +
// h) * R + row][split]; without lse_tag they go to l_ws as usual.
template <typename T>
struct PresetList {
  const int* k;  // read once wait() has returned
  T tok_k, tok_v;
  uint64_t* lse_tag;
  const uint32_t* epoch;  // read at the end
  const int* bad;
};
template <typename L>
struct is_preset : std::false_type {};
template <typename T>
struct is_preset<PresetList<T>> : std::true_type {};
struct SelectionRows {};
template <typename T, int D, int RTW, int MAXP, bool PAIR, bool COH, typename SeqLen, typename Wait,
          typename List = SelectionRows>
__device__ __forceinline__ void attend_role(const AttendArgs& a, int b, int h, int rg, int split,
                                            SeqLen&& seq_len_of, T* lds, int* s_phys, int* s_len,
                                            int* s_mask, int* s_tok, int tok_pos, Wait&& wait,
                                            List&& list) {
  using TL = Tiles<T, D>;
  const Geometry& g = a.g;
  const int bh = b * g.hk + h;
  const int nthreads = blockDim.x;
  const int tid = thread_index();
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6), nwaves = nthreads >> 6;
  const int ln16 = lane & 15, g4 = lane >> 4;

  // ---- per-row-tile state -------------------------------------------------
  // Q^T operand: lane holds row (rt*16 + ln16), d elements [kk*32 + 8*g4, +8)
  // (bf16) or [kq*16 + 4*g4, +4) (f32).
  constexpr int QREGS = (sizeof(T) == 2) ? D / 32 : D / 16;
  typedef typename std::conditional<sizeof(T) == 2, bf16x8, f32x4>::type qvec_t;
  qvec_t qop[RTW][QREGS];
  f32x4 acc[RTW][D / 16];
  float m_run[RTW], l_run[RTW];
  int row_r[RTW], row_tau[RTW];
  bool row_live[RTW];
  const int W = g.W;
#pragma unroll
  for (int j = 0; j < RTW; ++j) {
    const int lt = wave + j * nwaves;
    const int rt = rg * g.tiles_per_group + lt;
    const int rho = rt * 16 + ln16;
    const bool live = lt < g.tiles_per_group && rt < g.row_tiles && rho < g.R;
    const int r = live ? rho / g.G : 0;
    const int gq = live ? rho - r * g.G : 0;
    const int tau = a.step - W + r;
    row_r[j] = r;
    row_tau[j] = tau;
    row_live[j] = live && tau >= 0;
    m_run[j] = -INFINITY;
    l_run[j] = 0.f;
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) acc[j][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    const T* qrow = reinterpret_cast<const T*>(a.q) +
                    (((int64_t)b * (W + 1) + r) * g.hq + (int64_t)h * g.G + gq) * D;
#pragma unroll
    for (int kk = 0; kk < QREGS; ++kk) {
      if constexpr (sizeof(T) == 2) {
        bf16x8 v;
        if (live) {
          v = *reinterpret_cast<const bf16x8*>(qrow + kk * 32 + 8 * g4);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] = (__bf16)0.f;
        }
        qop[j][kk] = v;
      } else {
        f32x4 v = f32x4{0.f, 0.f, 0.f, 0.f};
        if (live) v = *reinterpret_cast<const f32x4*>(qrow + kk * 16 + 4 * g4);
        qop[j][kk] = v;
      }
    }
  }
  wait();
  // The split's rows of the selection are requested together with the number
  // of selected pages (slots past it hold -1 and are dropped below); thread i
  // handles slot i (kMaxSplitPages <= workgroup size).
  const int first = split * g.pages_per_split;
  int lp = -1, m = 0, phys = -1;
  int k_eff;
  constexpr bool kPreset = is_preset<typename std::decay<List>::type>::value;
  if constexpr (std::is_same<typename std::decay<List>::type, SelectionRows>::value) {
    if (tid < g.pages_per_split && first + tid < g.k_max) {
      const int64_t o = (int64_t)bh * g.k_max + first + tid;
      lp = get_c<COH>(a.sel + o);
      m = get_c<COH>(a.msk + o);
      if (a.sel_phys) phys = get_c<COH>(a.sel_phys + o);
    }
    k_eff = get_c<COH>(a.nsel + bh);
  } else if constexpr (kPreset) {
    k_eff = *list.k;
  } else {
    k_eff = list(tid, first, lp, m, phys);
  }
  const int seq_len = seq_len_of();
  const int np = min(g.pages_per_split, k_eff - first);
  // A split with nothing selected still writes its (empty) partial: (0, -inf)
  // for every row, so that the combine reads every split without first
  // reading the selection count.
  if (np > 0) {  // uniform
    const int nchunks = (np + g.chunk_pages - 1) / g.chunk_pages;
    // page list of the split: physical page (-1: skip), stored tokens (0 for a
    // skipped page and past the list), mask value
    if constexpr (!kPreset) {
      if (tid < kMaxSplitPages) {
        if (!a.sel_phys && tid < np && lp >= 0 && lp < g.max_pages)
          phys = a.pt[(int64_t)b * g.max_pages + lp];
        if (tid >= np || lp < 0 || lp >= g.max_pages || phys < 0 || phys >= g.num_phys) phys = -1;
        s_phys[tid] = phys;
        s_len[tid] = phys >= 0 ? max(0, min(g.P, seq_len - lp * g.P)) : 0;
        s_mask[tid] = tid < np ? m : 0;
        // the list slot of the step's token page, if it is in this split
        const uint64_t tm = wave_ballot(tok_pos >= 0 && phys >= 0 && lp == tok_pos / g.P);
        if (tid == 0) *s_tok = tm ? __builtin_ctzll(tm) : -1;
      }
      __syncthreads();  // page list ready
    }
    const int ts = *s_tok;
    T tok_kv[2];
    if constexpr (kPreset) {
      tok_kv[0] = list.tok_k;
      tok_kv[1] = list.tok_v;
    } else if (ts >= 0 && tid < D) {  // uniform condition, then the first D threads
      const int64_t o = ((int64_t)b * g.hk + h) * D + tid;
      tok_kv[0] = reinterpret_cast<const T*>(a.tok_k)[o];
      tok_kv[1] = reinterpret_cast<const T*>(a.tok_v)[o];
    }
    // Overwrite the token's key row and value column in LDS buffer `buf`, which
    // holds chunk c (after the barrier that follows its staging), then barrier.
    auto patch_token = [&](int c, int buf) {
      if (ts < 0 || ts / g.chunk_pages != c) return;  // uniform
      T* base = lds + buf * TL::BUF_ELEMS;
      const int row = (g.chunk_pages == 2 ? (ts & 1) * 16 : 0) + tok_pos % g.P;
      if (tid < D) {
        base[row * TL::KROW + tid] = tok_kv[0];
        base[TL::K_ELEMS + ((row >> 4) * D + tid) * TL::VROW + (row & 15)] = tok_kv[1];
      }
      __syncthreads();
    };

    // ---- chunk staging: global -> registers -> LDS ----------------------------
    const int pieces_per_thread = (TL::PIECES + nthreads - 1) / nthreads;
    // Chunks whose loads are in flight ahead of the computation: two when a
    // wavefront owns one row tile, one when it owns two (register budget).
    constexpr int DEPTH = RTW == 1 ? 2 : 1;
    uint4 stage[DEPTH][MAXP];
    const T* kc = reinterpret_cast<const T*>(a.kc);
    const T* vc = reinterpret_cast<const T*>(a.vc);

    // The part of each piece's address that does not depend on the chunk: its
    // 16-token tile (page of the chunk), its slot in the page, its element offset
    // in the page's (h_k) block and whether it is a V^T piece.  Page blocks of K
    // and V^T have the same size, P * d elements.
    int pc_tile[MAXP], pc_slot[MAXP], pc_off[MAXP];
    bool pc_v[MAXP];
  #pragma unroll
    for (int i = 0; i < MAXP; ++i) {
      const int e = min(tid + i * nthreads, TL::PIECES - 1);
      int tile, slot, off;
      const bool isv = e >= TL::K_PIECES;
      if (!isv) {
        const int tok = e / TL::KPR, q = e - tok * TL::KPR;
        tile = tok >> 4;
        slot = tok & 15;
        off = q * TL::VEC;  // + slot * D below
      } else {
        const int ev = e - TL::K_PIECES;
        tile = ev / (D * TL::VPR);
        const int rem = ev - tile * (D * TL::VPR);
        const int dr = rem / TL::VPR, q = rem - dr * TL::VPR;
        slot = q * TL::TPP;
        off = dr * g.P;  // + slot below
      }
      if (g.chunk_pages == 1) slot += 16 * tile;  // both tiles lie in one page
      pc_tile[i] = tile;
      pc_slot[i] = slot;
      pc_off[i] = isv ? off + slot : off + slot * D;
      pc_v[i] = isv;
    }

    // Every piece is loaded without a branch around the load (a piece that holds
    // no stored data reads the dummy line instead), so the loads of a chunk are
    // all in flight together; `keep` records how many
    // leading elements of each piece hold stored data (4 bits per piece), and
    // the rest is zeroed when the piece is written to LDS.
    const int64_t blk_elems = (int64_t)g.P * D;
    auto load_chunk = [&](int c, uint4* stage, uint32_t& keep) {
      uint32_t kp = 0u;
  #pragma unroll
      for (int i = 0; i < MAXP; ++i) {
        const int pl = g.chunk_pages == 2 ? 2 * c + pc_tile[i] : c;
        const int phys = s_phys[pl];
        const int len = s_len[pl];
        int n_el = pc_v[i] ? min(max(len - pc_slot[i], 0), TL::TPP) : (pc_slot[i] < len ? TL::VEC : 0);
        if (i >= pieces_per_thread || tid + i * nthreads >= TL::PIECES) n_el = 0;
        const T* src = reinterpret_cast<const T*>(a.dummy);
        if (n_el > 0)
          src = (pc_v[i] ? vc : kc) + ((int64_t)phys * g.hk + h) * blk_elems + pc_off[i];
        stage[i] = *reinterpret_cast<const uint4*>(src);
        kp |= (uint32_t)n_el << (4 * i);
      }
      keep = kp;
    };

    auto store_chunk = [&](int buf, const uint4* stage, uint32_t keep) {
      T* base = lds + buf * TL::BUF_ELEMS;
  #pragma unroll
      for (int i = 0; i < MAXP; ++i) {
        const int e = tid + i * nthreads;
        if (i < pieces_per_thread && e < TL::PIECES) {
          T* dst;
          if (e < TL::K_PIECES) {
            const int tok = e / TL::KPR, q = e - tok * TL::KPR;
            dst = base + tok * TL::KROW + q * TL::VEC;
          } else {
            const int ev = e - TL::K_PIECES;
            const int tile = ev / (D * TL::VPR);
            const int rem = ev - tile * (D * TL::VPR);
            const int dr = rem / TL::VPR, q = rem - dr * TL::VPR;
            dst = base + TL::K_ELEMS + (tile * D + dr) * TL::VROW + q * TL::TPP;
          }
          const int n_el = (keep >> (4 * i)) & 15;
          uint32_t w[4] = {stage[i].x, stage[i].y, stage[i].z, stage[i].w};
  #pragma unroll
          for (int t = 0; t < 4; ++t) {
            if constexpr (sizeof(T) == 2) {
              const uint32_t m = (2 * t < n_el ? 0x0000FFFFu : 0u) | (2 * t + 1 < n_el ? 0xFFFF0000u : 0u);
              w[t] &= m;
            } else {
              w[t] = t < n_el ? w[t] : 0u;
            }
          }
          *reinterpret_cast<uint4*>(dst) = make_uint4(w[0], w[1], w[2], w[3]);
        }
      }
    };

    // Attention over a group of NC chunks held in LDS (chunk c + i in buffer
    // (buf0 + i) & 1; only the first nv hold data): S for all of the group's
    // 16-token tiles, one online-softmax update over them, then O += P V per
    // chunk.  Grouping two chunks gives each wavefront twice the independent
    // matrix products per softmax step.
    auto compute_group = [&](auto nc_tag, int c, int buf0, int nv) {
      constexpr int NC = decltype(nc_tag)::value;
      constexpr int NT = 2 * NC;  // tiles of the group
      const T* Ks[NC];
      const T* Vs[NC];
  #pragma unroll
      for (int i = 0; i < NC; ++i) {
        Ks[i] = lds + ((buf0 + i) & 1) * TL::BUF_ELEMS;
        Vs[i] = Ks[i] + TL::K_ELEMS;
      }

      // page facts of the group's tiles: stored tokens from the tile's first
      // slot (0 past the group's valid chunks), mask value
      int tlen[NT], tmask[NT];
  #pragma unroll
      for (int tt = 0; tt < NT; ++tt) {
        const int cc = c + tt / 2, tile = tt & 1;
        const int pl = g.chunk_pages == 2 ? 2 * cc + tile : cc;
        const int so = g.chunk_pages == 2 ? 0 : 16 * tile;
        const bool in = tt / 2 < nv;
        tlen[tt] = in ? s_len[pl] - so : 0;
        tmask[tt] = in ? s_mask[pl] : 0;
      }

  #pragma unroll
      for (int j = 0; j < RTW; ++j) {
        const int lt = wave + j * nwaves;
        if (lt >= g.tiles_per_group || rg * g.tiles_per_group + lt >= g.row_tiles) break;  // uniform

        // ---- S^T = K . Q^T for every tile of the group
        f32x4 s[NT];
  #pragma unroll
        for (int tt = 0; tt < NT; ++tt) {
          f32x4 sacc = f32x4{0.f, 0.f, 0.f, 0.f};
          if (tt / 2 < nv) {  // uniform
            const T* krow = Ks[tt / 2] + ((tt & 1) * 16 + ln16) * TL::KROW;
            if constexpr (sizeof(T) == 2) {
  #pragma unroll
              for (int kk = 0; kk < D / 32; ++kk) {
                const bf16x8 kv = *reinterpret_cast<const bf16x8*>(krow + kk * 32 + 8 * g4);
                sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kv, qop[j][kk], sacc, 0, 0, 0);
              }
            } else {
  #pragma unroll
              for (int kq = 0; kq < D / 16; ++kq) {
                const f32x4 kv = *reinterpret_cast<const f32x4*>(krow + kq * 16 + 4 * g4);
  #pragma unroll
                for (int e = 0; e < 4; ++e)
                  sacc = __builtin_amdgcn_mfma_f32_16x16x4f32(kv[e], qop[j][kq][e], sacc, 0, 0, 0);
              }
            }
          }
          s[tt] = sacc;
        }

        // ---- mask, scale, online softmax (this lane: row ln16 of the tile)
        float x[NT][4];
        float mloc = -INFINITY;
  #pragma unroll
        for (int tt = 0; tt < NT; ++tt) {
          const bool use = row_live[j] && tlen[tt] > 0 &&
                           (row_r[j] == W || tmask[tt] < row_tau[j]);
  #pragma unroll
          for (int i = 0; i < 4; ++i) {
            const bool ok = use && (4 * g4 + i) < tlen[tt];
            x[tt][i] = ok ? s[tt][i] * a.scale_log2 : -INFINITY;
            mloc = fmaxf(mloc, x[tt][i]);
          }
        }
        mloc = col_max4(mloc);
        const float m_new = fmaxf(m_run[j], mloc);
        const float mu = (m_new == -INFINITY) ? 0.f : m_new;
        // the hardware exp2 (v_exp_f32, ~1 ulp): arguments are <= 0, and a
        // result below the normal range (a weight under 2^-126 of the row's
        // largest) becomes 0 instead of a denormal
        const float alpha = __builtin_amdgcn_exp2f(m_run[j] - mu);
        float p[NT][4];
        float psum = 0.f;
  #pragma unroll
        for (int tt = 0; tt < NT; ++tt)
  #pragma unroll
          for (int i = 0; i < 4; ++i) {
            p[tt][i] = __builtin_amdgcn_exp2f(x[tt][i] - mu);
            psum += p[tt][i];
          }
        l_run[j] = l_run[j] * alpha + psum;
        m_run[j] = m_new;
  #pragma unroll
        for (int dt = 0; dt < D / 16; ++dt) acc[j][dt] *= alpha;

        // ---- O^T += V^T . P^T, chunk by chunk
  #pragma unroll
        for (int i = 0; i < NC; ++i) {
          if (i >= nv) break;  // uniform
          if constexpr (sizeof(T) == 2) {
            bf16x8 ph, pl;
  #pragma unroll
            for (int e = 0; e < 8; ++e) {
              const float pv = p[2 * i + (e >> 2)][e & 3];
              const __bf16 hi = (__bf16)pv;
              ph[e] = hi;
              pl[e] = (__bf16)(pv - (float)hi);
            }
  #pragma unroll
            for (int dt = 0; dt < D / 16; ++dt) {
              const int dr = dt * 16 + ln16;
              const bf16x4 v0 = *reinterpret_cast<const bf16x4*>(Vs[i] + dr * TL::VROW + 4 * g4);
              const bf16x4 v1 = *reinterpret_cast<const bf16x4*>(Vs[i] + (D + dr) * TL::VROW + 4 * g4);
              const bf16x8 va = __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7);
              acc[j][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, ph, acc[j][dt], 0, 0, 0);
              acc[j][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, pl, acc[j][dt], 0, 0, 0);
            }
          } else {
  #pragma unroll
            for (int dt = 0; dt < D / 16; ++dt) {
              const int dr = dt * 16 + ln16;
  #pragma unroll
              for (int tile = 0; tile < 2; ++tile) {
                const f32x4 vv =
                    *reinterpret_cast<const f32x4*>(Vs[i] + (tile * D + dr) * TL::VROW + 4 * g4);
  #pragma unroll
                for (int e = 0; e < 4; ++e)
                  acc[j][dt] = __builtin_amdgcn_mfma_f32_16x16x4f32(vv[e], p[2 * i + tile][e],
                                                                   acc[j][dt], 0, 0, 0);
              }
            }
          }
        }
      }
    };
    auto compute_chunk = [&](int c, int buf) {
      compute_group(std::integral_constant<int, 1>{}, c, buf, 1);
    };

    // Chunk c goes through LDS buffer c & 1.  That buffer was last read while
    // computing chunk c - 2, and every wavefront has since passed the barrier of
    // chunk c - 1, so it can be rewritten.  Staging registers are indexed with
    // compile-time constants (two chunks per trip when DEPTH == 2).
    uint32_t keep[DEPTH];
    if constexpr (PAIR && DEPTH == 2) {
      // chunks in pairs: both of a pair in LDS and computed together while the
      // next pair's loads are in flight
      load_chunk(0, stage[0], keep[0]);
      if (nchunks > 1) load_chunk(1, stage[1], keep[1]);
  #pragma unroll 1
      for (int c = 0; c < nchunks; c += 2) {
        const int nv = min(2, nchunks - c);
        store_chunk(0, stage[0], keep[0]);
        if (nv > 1) store_chunk(1, stage[1], keep[1]);
        if (c + 2 < nchunks) load_chunk(c + 2, stage[0], keep[0]);
        if (c + 3 < nchunks) load_chunk(c + 3, stage[1], keep[1]);
        __syncthreads();
        patch_token(c, 0);
        if (nv > 1) patch_token(c + 1, 1);
        compute_group(std::integral_constant<int, 2>{}, c, 0, nv);
        if (c + 2 < nchunks) __syncthreads();  // the buffers are rewritten next trip
      }
    } else if constexpr (DEPTH == 2) {
      load_chunk(0, stage[0], keep[0]);
      if (nchunks > 1) load_chunk(1, stage[DEPTH - 1], keep[DEPTH - 1]);
  #pragma unroll 1
      for (int c = 0; c < nchunks; c += 2) {
        store_chunk(0, stage[0], keep[0]);
        if (c + 2 < nchunks) load_chunk(c + 2, stage[0], keep[0]);
        __syncthreads();
        patch_token(c, 0);
        compute_chunk(c, 0);
        if (c + 1 < nchunks) {
          store_chunk(1, stage[DEPTH - 1], keep[DEPTH - 1]);
          if (c + 3 < nchunks) load_chunk(c + 3, stage[DEPTH - 1], keep[DEPTH - 1]);
          __syncthreads();
          patch_token(c + 1, 1);
          compute_chunk(c + 1, 1);
        }
      }
    } else {
      load_chunk(0, stage[0], keep[0]);
  #pragma unroll 1
      for (int c = 0; c < nchunks; ++c) {
        store_chunk(c & 1, stage[0], keep[0]);
        if (c + 1 < nchunks) load_chunk(c + 1, stage[0], keep[0]);
        __syncthreads();
        patch_token(c, c & 1);
        compute_chunk(c, c & 1);
      }
    }
  }

  // ---- normalise and write this split's partial (O, LSE) per row -------------
  const int64_t part = ((int64_t)bh * g.n_splits + split) * g.R;
#pragma unroll
  for (int j = 0; j < RTW; ++j) {
    const int lt = wave + j * nwaves;
    const int rt = rg * g.tiles_per_group + lt;
    if (lt >= g.tiles_per_group || rt >= g.row_tiles) break;
    const float l = col_sum4(l_run[j]);
    const int rho = rt * 16 + ln16;
    if (rho < g.R) {
      const float inv = l > 0.f ? 1.f / l : 0.f;
      float* orow = a.o_ws + (part + rho) * D;
      const float lse = l > 0.f ? (m_run[j] + __log2f(l)) * kLn2 : -INFINITY;
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) {
        const f32x4 o = acc[j][dt] * inv;
        if constexpr (COH) {
          const uint32_t off = (uint32_t)(((part + rho) * D + dt * 16 + 4 * g4) * sizeof(float));
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4v, o),
                                                 coherent_rsrc(a.o_ws), off, 0, kCpolSc1);
        } else {
          // streamed out: read once by the combine, not worth keeping in L2
          __builtin_nontemporal_store(o, reinterpret_cast<f32x4*>(orow + dt * 16 + 4 * g4));
        }
      }
      if constexpr (COH && is_preset<typename std::decay<List>::type>::value) {
        if (list.lse_tag) {
          // the row's output words are acknowledged (written through) before
          // its tag goes out: a reader that sees the tag finds them
          __builtin_amdgcn_s_waitcnt(0);
          if (g4 == 0) {
            const uint64_t hi = (uint64_t)(*list.epoch | (*list.bad ? 0x80000000u : 0u)) << 32;
            __hip_atomic_store(list.lse_tag + ((int64_t)bh * g.R + rho) * g.n_splits + split,
                               hi | __float_as_uint(lse), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          }
        } else if (g4 == 0) {
          a.l_ws[part + rho] = lse;
        }
      } else if (g4 == 0) {
        if constexpr (COH) put_c<true>(a.l_ws + part + rho, lse);
        else __builtin_nontemporal_store(lse, a.l_ws + part + rho);
      }
    }
  }
}

// ============================================================================
// Combine + merge role (see merge.hip for the design).
// ============================================================================
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
  int32_t* seq_lens;    // advanced past a pending token (Geometry::token_pending), or null
  const int32_t* pt;
  // last_loaded update of the step (Alg. 2) when the selection was made without
  // it: the kept pages (selection rows, counts) get the step, the token page
  // tok_upd[bh] (-1: none) step - 1.  Null: no update.
  int32_t* a_upd;
  const int32_t* sel_upd;
  const int32_t* tok_upd;
  // sticky error word of the launch that produced the partials (a bounded wait
  // ran out there), or null: when set, the rows are written as NaN
  const int32_t* err;
};

template <int D>
struct Row {
  static constexpr int E = D / 64;
  float o[E];
  float z;
};

// Combine the splits of NR rows rho[] of (b, h): sum_s e^{Z_s} O_s / sum_s e^{Z_s},
// Z = ln sum_s e^{Z_s}.  Splits are taken GS at a time with every load of the
// group (log-normalisers one per lane, output rows E floats per lane) in
// flight together; groups after the first are folded in relative to the
// running maximum.
// COH: the partials and the selection count come from other workgroups of the
// same launch: device-coherent loads.  ZPRE: the log-normalisers are not loaded
// here: lane s of zl.z[r] holds split s's for row r (at most 64 splits).
struct ZLanes {
  float z[2];
};
template <int D, int NR, int GS, bool COH, bool ZPRE = false>
__device__ __forceinline__ void combine_splits(const MergeArgs& a, int bh, const int (&rho)[NR],
                                               Row<D> (&res)[NR], const ZLanes& zl) {
  constexpr int E = Row<D>::E;
  const Geometry& g = a.g;
  const int lane = thread_index() & 63;
  const int e0 = lane * E;
  // every split holds a partial, (0, -inf) if nothing was selected in it
  const int nvs = g.n_splits;
  float m[NR], wl[NR], acc[NR][E];
#pragma unroll
  for (int r = 0; r < NR; ++r) {
    m[r] = -INFINITY;
    wl[r] = 0.f;
#pragma unroll
    for (int e = 0; e < E; ++e) acc[r][e] = 0.f;
  }
  for (int s0 = 0; s0 < nvs; s0 += GS) {
    const int cnt = min(GS, nvs - s0);
    float z[NR], v[NR][GS][E];
#pragma unroll
    for (int r = 0; r < NR; ++r) {
      const int64_t base = (int64_t)bh * g.n_splits * g.R + rho[r];
      if constexpr (ZPRE) {
        const float zs = s0 == 0 ? zl.z[r] : __shfl(zl.z[r], min(s0 + lane, 63));
        z[r] = lane < cnt ? zs : -INFINITY;
      } else {
        z[r] = lane < cnt ? get_c<COH>(a.l_ws + base + (int64_t)(s0 + lane) * g.R) : -INFINITY;
      }
      // E == 2: split s0 + j's row at byte offset o_j = o_0 + j * stride in
      // the head's block of partial rows (uniform: the scalar offset of the
      // load, the lane's part the vector one), clamped to the group's last
      // split; two scalar operations a row.  The host keeps a head's block
      // below 2 GiB.
      const float* hblk = a.o_ws + (int64_t)bh * g.n_splits * g.R * D;
      const uint32_t stride = (uint32_t)(g.R * D * sizeof(float));
      uint32_t o = (uint32_t)(((int64_t)s0 * g.R + rho[r]) * D * sizeof(float));
      const uint32_t o_last = o + (uint32_t)(cnt - 1) * stride;
#pragma unroll
      for (int j = 0; j < GS; ++j) {
        const int64_t row = base + (int64_t)(s0 + min(j, cnt - 1)) * g.R;
        if constexpr (E == 2) {
          const u32x2 w = __builtin_amdgcn_raw_buffer_load_b64(
              coherent_rsrc(hblk), (uint32_t)(e0 * sizeof(float)), min(o, o_last),
              COH ? kCpolSc1 : 0);
          o += stride;
          v[r][j][0] = __uint_as_float(w[0]);
          v[r][j][1] = __uint_as_float(w[1]);
        } else {
#pragma unroll
          for (int e = 0; e < E; ++e) v[r][j][e] = get_c<COH>(a.o_ws + row * D + e0 + e);
        }
      }
    }
#pragma unroll
    for (int r = 0; r < NR; ++r) {
      const float m_new = fmaxf(m[r], wave_max(z[r]));
      if (m_new == -INFINITY) continue;  // uniform: no split holds a selected entry yet
      const float scale = __expf(m[r] - m_new);  // 0 while m is -inf
      wl[r] *= scale;
#pragma unroll
      for (int e = 0; e < E; ++e) acc[r][e] *= scale;
      const float w = lane < cnt ? __expf(z[r] - m_new) : 0.f;
      wl[r] += w;
#pragma unroll
      for (int j = 0; j < GS; ++j) {
        const float wj = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(w), j));
#pragma unroll
        for (int e = 0; e < E; ++e) acc[r][e] += wj * v[r][j][e];  // wj = 0 past cnt
      }
      m[r] = m_new;
    }
  }
#pragma unroll
  for (int r = 0; r < NR; ++r) {
    if (m[r] == -INFINITY) {
#pragma unroll
      for (int e = 0; e < E; ++e) res[r].o[e] = 0.f;
      res[r].z = -INFINITY;
      continue;
    }
    const float wsum = wave_sum(wl[r]);
    const float inv = 1.f / wsum;
#pragma unroll
    for (int e = 0; e < E; ++e) res[r].o[e] = acc[r][e] * inv;
    res[r].z = m[r] + __logf(wsum);
  }
}

template <int D>
__device__ __forceinline__ Row<D> lse_merge(const Row<D>& x, const Row<D>& y) {
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
__device__ __forceinline__ void put(float* o, float* z, int64_t idx, const Row<D>& v) {
  const int e0 = (thread_index() & 63) * Row<D>::E;
#pragma unroll
  for (int e = 0; e < Row<D>::E; ++e) o[idx * D + e0 + e] = v.o[e];
  if ((thread_index() & 63) == 0) z[idx] = v.z;
}

template <int D>
__device__ __forceinline__ Row<D> get(const float* o, const float* z, int64_t idx) {
  Row<D> v;
  const int e0 = (thread_index() & 63) * Row<D>::E;
#pragma unroll
  for (int e = 0; e < Row<D>::E; ++e) v.o[e] = o[idx * D + e0 + e];
  v.z = z[idx];
  return v;
}

// The partial (O, Z) of window rows r[] of query head gq of (b, h): from the
// split partials, or (mode 1) from the caller's o_part / lse_part.
template <int D, int NR, int GS, bool COH, bool ZPRE = false>
__device__ __forceinline__ void partials(const MergeArgs& a, int b, int h, int gq, const int (&r)[NR],
                                         Row<D> (&res)[NR], const ZLanes& zl) {
  const Geometry& g = a.g;
  if (a.mode == 1) {
#pragma unroll
    for (int i = 0; i < NR; ++i)
      res[i] = get<D>(a.o_part, a.l_part, ((int64_t)b * (g.W + 1) + r[i]) * g.hq + h * g.G + gq);
    return;
  }
  int rho[NR];
#pragma unroll
  for (int i = 0; i < NR; ++i) rho[i] = r[i] * g.G + gq;
  combine_splits<D, NR, GS, COH, ZPRE>(a, b * g.hk + h, rho, res, zl);
}

// Where merge unit `unit` = ((b * h_k + h) * G + gq) * xs + x works: window
// row x of query head gq of (sequence b, KV head h).
struct UnitPos {
  int x, gq, h, b;
};
__device__ __forceinline__ UnitPos unit_pos(const MergeArgs& a, int unit) {
  const Geometry& g = a.g;
  int u = unit;
  const int x = u % a.xs;
  u /= a.xs;
  const int gq = u % g.G;
  u /= g.G;
  return UnitPos{x, gq, u % g.hk, u / g.hk};
}

// The output-cache row the merge unit at p merges its partial with (see
// merge_unit), or -1 if it has none: row x > 0 of a step whose query exists,
// and for x = 0 the slot of the row leaving the window.
__device__ __forceinline__ int64_t unit_cache_row(const MergeArgs& a, const UnitPos& p) {
  const Geometry& g = a.g;
  const int W = g.W;
  if (a.mode == 0 || p.x == W) return -1;
  const int tau0 = a.step - W + p.x;
  if (tau0 < 0) return -1;
  const int slot = p.x > 0 ? tau0 % W : a.step % W;  // (t - W) mod W == t mod W
  return ((int64_t)p.b * W + slot) * g.hq + p.h * g.G + p.gq;
}

// One work unit of the combine + merge: unit = ((b * h_k + h) * G + gq) * xs + x,
// executed by one wavefront; no barriers inside.  The unit of row 0 also
// handles the current row W, whose cache slot is the one row 0 leaves.  GS:
// splits whose loads are in flight together (at most 64).  ZPRE: the splits'
// log-normalisers of the unit's rows (x, then W for x == 0 < W) are in zl.
// PRE: `pre` is the row unit_cache_row names, loaded by the caller (it may
// load it early: no other unit reads or writes it), instead of here.
template <int D, int GS, bool COH = false, bool ZPRE = false, bool PRE = false>
__device__ __forceinline__ void merge_unit(const MergeArgs& a, const UnitPos& up,
                                           const ZLanes& zl = ZLanes{}, Row<D> pre = Row<D>{}) {
  const Geometry& g = a.g;
  const int W = g.W;
  const int x = up.x, gq = up.gq, h = up.h, b = up.b;
  const int qh = h * g.G + gq;
  const int64_t out_row = (int64_t)b * (W + 1);

  if (a.mode == 0 || x == W) {  // plain combine of row x (W == 0: the current row only)
    Row<D> p[1];
    partials<D, 1, GS, COH, ZPRE>(a, b, h, gq, {x}, p, zl);
    if (a.mode == 0)
      put<D>(a.o_part_out, a.l_part_out, (out_row + x) * g.hq + qh, p[0]);
    else
      put<D>(a.o_out, a.l_out, (out_row + x) * g.hq + qh, p[0]);
    return;
  }

  const int tau0 = a.step - W + x;
  Row<D> zero;
#pragma unroll
  for (int e = 0; e < Row<D>::E; ++e) zero.o[e] = 0.f;
  zero.z = -INFINITY;
  if (x > 0) {
    if (tau0 < 0) {  // the row's query does not exist yet
      put<D>(a.o_out, a.l_out, (out_row + x) * g.hq + qh, zero);
      return;
    }
    const int64_t ci = ((int64_t)b * W + tau0 % W) * g.hq + qh;
    const Row<D> cached = PRE ? pre : get<D>(a.o_cache, a.l_cache, ci);
    Row<D> p[1];
    partials<D, 1, GS, COH, ZPRE>(a, b, h, gq, {x}, p, zl);
    const Row<D> merged = lse_merge<D>(cached, p[0]);
    put<D>(a.o_cache, a.l_cache, ci, merged);
    put<D>(a.o_out, a.l_out, (out_row + x) * g.hq + qh, merged);
    return;
  }
  // Row 0 leaves the window (final); the current row then takes its slot,
  // (t - W) mod W == t mod W.
  const int64_t slot = ((int64_t)b * W + a.step % W) * g.hq + qh;
  Row<D> cached = zero;
  if (tau0 >= 0) cached = PRE ? pre : get<D>(a.o_cache, a.l_cache, slot);
  Row<D> p[2];
  partials<D, 2, GS, COH, ZPRE>(a, b, h, gq, {0, W}, p, zl);
  const Row<D> merged = tau0 >= 0 ? lse_merge<D>(cached, p[0]) : zero;
  put<D>(a.o_out, a.l_out, out_row * g.hq + qh, merged);
  put<D>(a.o_out, a.l_out, (out_row + W) * g.hq + qh, p[1]);
  // the slot's old contents are in registers (merged depends on them) before
  // it is overwritten
  asm volatile("" : : "v"(merged.z) : "memory");
  put<D>(a.o_cache, a.l_cache, slot, p[1]);
}

// The output rows merge unit `unit` writes, as NaN; nothing else is written
// (the output cache keeps its rows).
template <int D>
__device__ __forceinline__ void poison_unit(const MergeArgs& a, const UnitPos& up) {
  const Geometry& g = a.g;
  const int x = up.x, gq = up.gq, h = up.h, b = up.b;
  const int qh = h * g.G + gq;
  const int64_t out_row = (int64_t)b * (g.W + 1);
  Row<D> p;
#pragma unroll
  for (int e = 0; e < Row<D>::E; ++e) p.o[e] = __builtin_nanf("");
  p.z = __builtin_nanf("");
  put<D>(a.o_out, a.l_out, (out_row + x) * g.hq + qh, p);
  if (x == 0 && g.W > 0) put<D>(a.o_out, a.l_out, (out_row + g.W) * g.hq + qh, p);
}

MergeArgs make_merge_args(const Geometry& g, int step, int mode, const float* o_ws,
                          const float* l_ws, const int32_t* num_selected, const float* o_part,
                          const float* l_part, float* o_part_out, float* l_part_out,
                          const retro_output_cache* oc, float* o_out, float* lse_out);

}  // namespace retro
