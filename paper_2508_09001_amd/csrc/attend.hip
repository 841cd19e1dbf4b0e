// One attention pass over the selected pages for the W+1 queries of the
// retrospective window (Alg. 1 "Attention"; eq. update-org for the current
// query, eq. update-sup for the past ones, masked as in the "Retrospective Mask"
// paragraph: row tau uses page p iff tau == t or M_p < tau).
//
// Work decomposition.  A workgroup owns one (sequence, KV head, split), a split
// being a run of consecutive entries of the selected-page list, processed as
// 32-token chunks (two 16-token tiles: two pages of 16, or one page of 32).
// Every chunk's keys and values are read from HBM once, staged in LDS, and used
// by all R = (W+1)*G rows of the KV head's group (row = window step r times G
// plus query head), so the gather is shared by the whole window and group.
// Rows are split into 16-row tiles; each wavefront owns RTW row tiles.
//
// Per chunk and row tile, on MFMA (gfx950):
//   S^T (16 tokens x 16 rows) = K (16 x d) . Q^T (d x 16), per 16-token tile
//       bf16: v_mfma_f32_16x16x32_bf16, d/32 steps;  f32: 16x16x4, d/4 steps
//   masking, online softmax in registers (exp2 domain, running max per row)
//   O^T (16 d x 16 rows) += V^T (16 d x 32 tokens) . P^T (32 tokens x 16 rows)
//       bf16: P is split into bf16 hi + lo parts (two MFMAs) so that rounding P
//             to bf16 does not cost accuracy; f32: 16x16x4.
// The S^T accumulator layout (lane l: row l%16, tokens 4*(l/16)..+3) is exactly
// the B operand layout of the PV product once the 32 chunk tokens are ordered
// as [tile 0: 4g..4g+3, tile 1: 4g..4g+3] for lane group g; V^T is read from LDS
// in the same token order, so no data moves between lanes.  The running max is
// per row, i.e. per lane column, and the O^T accumulator keeps the row in the
// lane column too, so rescaling needs no shuffles.
//
// Values live d-major in the cache (v_cache[page][h][d][P]), which is what makes
// the PV operand a contiguous LDS read.
//
// Output: per split and row, the normalised partial output and its natural-log
// normaliser, combined across splits by the merge kernel.
#include "internal.h"

namespace retro {
namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kMaxPieces = 4;  // 16-byte staging registers per thread per chunk

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
};

template <typename T, int D, int RTW>
__global__ void __launch_bounds__(512) attend_kernel(AttendArgs a) {
  using TL = Tiles<T, D>;
  constexpr int NBUF = 2;
  constexpr int MAX_SPLIT_PAGES = 64;
  __shared__ __attribute__((aligned(16))) T lds[NBUF * TL::BUF_ELEMS];
  __shared__ int s_phys[MAX_SPLIT_PAGES];
  __shared__ int s_page[MAX_SPLIT_PAGES];
  __shared__ int s_mask[MAX_SPLIT_PAGES];

  const Geometry& g = a.g;
  // Work units are ordered (sequence, KV head, row group, split), split fastest,
  // and spread so that the units of one KV head share an XCD (workgroups go to
  // the 8 XCDs round-robin): its partial outputs then stay in that XCD's L2 for
  // the combine.
  int u = xcd_remap(blockIdx.x, gridDim.x);
  const int split = u % g.n_splits;
  u /= g.n_splits;
  const int rg = u % g.n_rgroups;
  u /= g.n_rgroups;
  const int h = u % g.hk, b = u / g.hk;
  const int bh = b * g.hk + h;
  const int k_eff = a.nsel[bh];
  const int first = split * g.pages_per_split;
  const int np = min(g.pages_per_split, k_eff - first);
  if (np <= 0) return;  // uniform: nothing selected in this split
  const int seq_len = a.seq_lens[b];
  const int nthreads = blockDim.x;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, nwaves = nthreads >> 6;
  const int ln16 = lane & 15, g4 = lane >> 4;
  const int nchunks = (np + g.chunk_pages - 1) / g.chunk_pages;

  for (int i = tid; i < np; i += nthreads) {
    const int lp = a.sel[(int64_t)bh * g.k_max + first + i];
    int phys = -1;
    if (a.sel_phys) {
      phys = a.sel_phys[(int64_t)bh * g.k_max + first + i];
    } else if (lp >= 0 && lp < g.max_pages) {
      phys = a.pt[(int64_t)b * g.max_pages + lp];
    }
    if (lp < 0 || lp >= g.max_pages || phys < 0 || phys >= g.num_phys) phys = -1;
    s_phys[i] = phys;
    s_page[i] = lp;
    s_mask[i] = a.msk[(int64_t)bh * g.k_max + first + i];
  }

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
  __syncthreads();  // page list ready

  // ---- chunk staging: global -> registers -> LDS ----------------------------
  const int pieces_per_thread = (TL::PIECES + nthreads - 1) / nthreads;
  // Chunks whose loads are in flight ahead of the computation: two when a
  // wavefront owns one row tile, one when it owns two (register budget).
  constexpr int DEPTH = RTW == 1 ? 2 : 1;
  uint4 stage[DEPTH][kMaxPieces];
  const T* kc = reinterpret_cast<const T*>(a.kc);
  const T* vc = reinterpret_cast<const T*>(a.vc);

  auto tile_page = [&](int c, int tile, int* slot_off) -> int {
    // split-local page index of a 16-token tile of chunk c, and its slot offset
    if (g.chunk_pages == 2) {
      *slot_off = 0;
      return 2 * c + tile;
    }
    *slot_off = 16 * tile;
    return c;
  };

  auto load_chunk = [&](int c, uint4* stage) {
#pragma unroll
    for (int i = 0; i < kMaxPieces; ++i) {
      const int e = tid + i * nthreads;
      uint4 v = make_uint4(0u, 0u, 0u, 0u);
      if (i < pieces_per_thread && e < TL::PIECES) {
        if (e < TL::K_PIECES) {
          const int tok = e / TL::KPR, q = e - tok * TL::KPR;
          const int tile = tok >> 4;
          int so;
          const int pl = tile_page(c, tile, &so);
          const int slot = so + (tok & 15);
          if (pl < np && s_phys[pl] >= 0 && s_page[pl] * g.P + slot < seq_len) {
            const T* src = kc + (((int64_t)s_phys[pl] * g.hk + h) * g.P + slot) * D + q * TL::VEC;
            v = *reinterpret_cast<const uint4*>(src);
          }
        } else {
          const int ev = e - TL::K_PIECES;
          const int tile = ev / (D * TL::VPR);
          const int rem = ev - tile * (D * TL::VPR);
          const int dr = rem / TL::VPR, q = rem - dr * TL::VPR;
          int so;
          const int pl = tile_page(c, tile, &so);
          if (pl < np && s_phys[pl] >= 0) {
            const int slot0 = so + q * TL::TPP;
            const int valid = seq_len - (s_page[pl] * g.P + slot0);  // stored tokens in piece
            if (valid > 0) {
              const T* src = vc + (((int64_t)s_phys[pl] * g.hk + h) * D + dr) * g.P + slot0;
              v = *reinterpret_cast<const uint4*>(src);
              if (valid < TL::TPP) {  // zero the unstored tail of the piece
                uint32_t w[4] = {v.x, v.y, v.z, v.w};
                if constexpr (sizeof(T) == 2) {
#pragma unroll
                  for (int t = 0; t < 8; ++t)
                    if (t >= valid) w[t >> 1] &= (t & 1) ? 0x0000FFFFu : 0xFFFF0000u;
                } else {
#pragma unroll
                  for (int t = 0; t < 4; ++t)
                    if (t >= valid) w[t] = 0u;
                }
                v = make_uint4(w[0], w[1], w[2], w[3]);
              }
            }
          }
        }
      }
      stage[i] = v;
    }
  };

  auto store_chunk = [&](int buf, const uint4* stage) {
    T* base = lds + buf * TL::BUF_ELEMS;
#pragma unroll
    for (int i = 0; i < kMaxPieces; ++i) {
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
        *reinterpret_cast<uint4*>(dst) = stage[i];
      }
    }
  };

  auto compute_chunk = [&](int c, int buf) {
    const T* Ks = lds + buf * TL::BUF_ELEMS;
    const T* Vs = Ks + TL::K_ELEMS;

    // page facts for the two tiles of this chunk
    bool tvalid[2];
    int tmask[2], tbase[2];
#pragma unroll
    for (int tile = 0; tile < 2; ++tile) {
      int so;
      const int pl = tile_page(c, tile, &so);
      tvalid[tile] = pl < np && s_phys[pl] >= 0;
      tmask[tile] = tvalid[tile] ? s_mask[pl] : 0;
      tbase[tile] = tvalid[tile] ? s_page[pl] * g.P + so : 0;  // position of tile slot 0
    }

#pragma unroll
    for (int j = 0; j < RTW; ++j) {
      const int lt = wave + j * nwaves;
      if (lt >= g.tiles_per_group || rg * g.tiles_per_group + lt >= g.row_tiles) break;  // uniform

      // ---- S^T = K . Q^T for both tiles
      f32x4 s[2];
#pragma unroll
      for (int tile = 0; tile < 2; ++tile) {
        f32x4 sacc = f32x4{0.f, 0.f, 0.f, 0.f};
        const T* krow = Ks + (tile * 16 + ln16) * TL::KROW;
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
        s[tile] = sacc;
      }

      // ---- mask, scale, online softmax (this lane: row ln16 of the tile)
      float x[2][4];
      float mloc = -INFINITY;
#pragma unroll
      for (int tile = 0; tile < 2; ++tile) {
        const bool use = row_live[j] && tvalid[tile] &&
                         (row_r[j] == W || tmask[tile] < row_tau[j]);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const bool ok = use && (tbase[tile] + 4 * g4 + i) < seq_len;
          x[tile][i] = ok ? s[tile][i] * a.scale_log2 : -INFINITY;
          mloc = fmaxf(mloc, x[tile][i]);
        }
      }
      mloc = fmaxf(mloc, __shfl_xor(mloc, 16));
      mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
      const float m_new = fmaxf(m_run[j], mloc);
      const float mu = (m_new == -INFINITY) ? 0.f : m_new;
      const float alpha = exp2f(m_run[j] - mu);
      float p[2][4];
      float psum = 0.f;
#pragma unroll
      for (int tile = 0; tile < 2; ++tile)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          p[tile][i] = exp2f(x[tile][i] - mu);
          psum += p[tile][i];
        }
      l_run[j] = l_run[j] * alpha + psum;
      m_run[j] = m_new;
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) acc[j][dt] *= alpha;

      // ---- O^T += V^T . P^T
      if constexpr (sizeof(T) == 2) {
        bf16x8 ph, pl;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float pv = p[e >> 2][e & 3];
          const __bf16 hi = (__bf16)pv;
          ph[e] = hi;
          pl[e] = (__bf16)(pv - (float)hi);
        }
#pragma unroll
        for (int dt = 0; dt < D / 16; ++dt) {
          const int dr = dt * 16 + ln16;
          const bf16x4 v0 = *reinterpret_cast<const bf16x4*>(Vs + dr * TL::VROW + 4 * g4);
          const bf16x4 v1 = *reinterpret_cast<const bf16x4*>(Vs + (D + dr) * TL::VROW + 4 * g4);
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
            const f32x4 vv = *reinterpret_cast<const f32x4*>(Vs + (tile * D + dr) * TL::VROW + 4 * g4);
#pragma unroll
            for (int e = 0; e < 4; ++e)
              acc[j][dt] = __builtin_amdgcn_mfma_f32_16x16x4f32(vv[e], p[tile][e], acc[j][dt], 0, 0, 0);
          }
        }
      }
    }

  };

  // Chunk c goes through LDS buffer c & 1.  That buffer was last read while
  // computing chunk c - 2, and every wavefront has since passed the barrier of
  // chunk c - 1, so it can be rewritten.  Staging registers are indexed with
  // compile-time constants (two chunks per trip when DEPTH == 2).
  if constexpr (DEPTH == 2) {
    load_chunk(0, stage[0]);
    if (nchunks > 1) load_chunk(1, stage[DEPTH - 1]);
#pragma unroll 1
    for (int c = 0; c < nchunks; c += 2) {
      store_chunk(0, stage[0]);
      if (c + 2 < nchunks) load_chunk(c + 2, stage[0]);
      __syncthreads();
      compute_chunk(c, 0);
      if (c + 1 < nchunks) {
        store_chunk(1, stage[DEPTH - 1]);
        if (c + 3 < nchunks) load_chunk(c + 3, stage[DEPTH - 1]);
        __syncthreads();
        compute_chunk(c + 1, 1);
      }
    }
  } else {
    load_chunk(0, stage[0]);
#pragma unroll 1
    for (int c = 0; c < nchunks; ++c) {
      store_chunk(c & 1, stage[0]);
      if (c + 1 < nchunks) load_chunk(c + 1, stage[0]);
      __syncthreads();
      compute_chunk(c, c & 1);
    }
  }

  // ---- normalise and write this split's partial (O, LSE) per row -------------
  const int64_t part = ((int64_t)bh * g.n_splits + split) * g.R;
#pragma unroll
  for (int j = 0; j < RTW; ++j) {
    const int lt = wave + j * nwaves;
    const int rt = rg * g.tiles_per_group + lt;
    if (lt >= g.tiles_per_group || rt >= g.row_tiles) break;
    float l = l_run[j];
    l += __shfl_xor(l, 16);
    l += __shfl_xor(l, 32);
    const int rho = rt * 16 + ln16;
    if (rho < g.R) {
      const float inv = l > 0.f ? 1.f / l : 0.f;
      float* orow = a.o_ws + (part + rho) * D;
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) {
        const f32x4 o = acc[j][dt] * inv;
        *reinterpret_cast<f32x4*>(orow + dt * 16 + 4 * g4) = o;
      }
      if (g4 == 0) a.l_ws[part + rho] = l > 0.f ? (m_run[j] + __log2f(l)) * kLn2 : -INFINITY;
    }
  }
}

template <typename T, int D, int RTW>
hipError_t attend_t(const AttendArgs& a, hipStream_t s) {
  const Geometry& g = a.g;
  const int64_t n = (int64_t)g.n_splits * g.n_rgroups * g.hk * g.batch;
  attend_kernel<T, D, RTW><<<(unsigned)n, 64 * g.waves, 0, s>>>(a);
  return hipGetLastError();
}

template <typename T, int D>
hipError_t attend_d(const AttendArgs& a, hipStream_t s) {
  switch (a.g.rtw) {
    case 1: return attend_t<T, D, 1>(a, s);
    default: return attend_t<T, D, 2>(a, s);
  }
}

}  // namespace

int attend_min_waves(int dtype, int D) {
  const int pieces = dtype == RETRO_BF16 ? (D == 128 ? Tiles<bf16_t, 128>::PIECES : Tiles<bf16_t, 64>::PIECES)
                                         : (D == 128 ? Tiles<float, 128>::PIECES : Tiles<float, 64>::PIECES);
  return (pieces + 64 * kMaxPieces - 1) / (64 * kMaxPieces);
}

hipError_t launch_attend(const Geometry& g, int step, const void* q_window,
                         const retro_kv_cache& c, const retro_selection& sel,
                         const int32_t* sel_phys, float* o_ws, float* l_ws, hipStream_t s) {
  AttendArgs a;
  a.g = g;
  a.step = step;
  a.scale_log2 = g.sm_scale * kLog2e;
  a.q = q_window;
  a.kc = c.k_cache;
  a.vc = c.v_cache;
  a.pt = c.page_table;
  a.seq_lens = c.seq_lens;
  a.sel = sel.selected;
  a.msk = sel.mask;
  a.nsel = sel.num_selected;
  a.sel_phys = sel_phys;
  a.o_ws = o_ws;
  a.l_ws = l_ws;
  if (g.dtype == RETRO_BF16) return g.D == 128 ? attend_d<bf16_t, 128>(a, s) : attend_d<bf16_t, 64>(a, s);
  return g.D == 128 ? attend_d<float, 128>(a, s) : attend_d<float, 64>(a, s);
}

}  // namespace retro
