// Dense projections of the multi-layer decode with re-embedding (Sec. 3.3): the
// W+1 window rows of every sequence, a few dozen at most, times a weight matrix.
// With so few rows the product is bound by reading the weight once from HBM
// (the paper's appendix on linear layers makes the same point), so each weight is
// stored pre-tiled for the MFMA operand layout: one wavefront load of 1 KB per
// 16 columns x 32 reduction elements, contiguous in memory.
//
// Packed layout of a [K][N] weight (y = x . w): [N/16][K/32][4][16][8] bf16;
// element (k, n) sits at tile n/16, step k/32, group (k%32)/8, column n%16,
// position k%8.  Lane l = 16 * group + column of a wavefront then holds exactly
// the B operand of v_mfma_f32_16x16x32_bf16 for its column.
//
// A workgroup owns 16 output columns; its PJ_WAVES wavefronts split the
// reduction, each accumulating all row tiles (16 rows each) of its share with
// MFMA, and the shares are summed in a fixed order through LDS.  Sixteen
// wavefronts of 512 reduction elements each load their whole share of a
// 4096-deep weight in one pass: the launch is a single round trip to HBM per
// wavefront, which is what a few-row product costs.
#include <hip/hip_runtime.h>

#include "internal.h"
#include "proj.h"

namespace retro {
namespace {

constexpr int PJ_WAVES = 16;         // wavefronts per workgroup, each a slice of the reduction
constexpr int PJ_MIN_STEPS = 2;      // 32-element reduction steps per wavefront (at least)
constexpr int PJ_MAX_ROW_TILES = 7;  // up to 112 rows (more would spill registers)

__device__ __forceinline__ uint16_t bf16_rne(float x) {
  const uint32_t u = __float_as_uint(x);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0;  // NaN stays NaN
  return static_cast<uint16_t>((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

__device__ __forceinline__ bf16x8 bits_to_bf16x8(uint4 u) {
  return __builtin_bit_cast(bf16x8, u);
}

// A operand: row `row` of x, elements [k, k + 8); zero past the last row.
// x is bf16 [rows][K], or f32 [rows][K] rounded to bf16 here.
template <bool F32IN>
__device__ __forceinline__ bf16x8 load_a(const void* x, int rows, int K, int row, int k) {
  if (row >= rows) return bits_to_bf16x8(make_uint4(0, 0, 0, 0));
  if constexpr (F32IN) {
    const float* p = static_cast<const float*>(x) + (int64_t)row * K + k;
    const float4 lo = *reinterpret_cast<const float4*>(p);
    const float4 hi = *reinterpret_cast<const float4*>(p + 4);
    uint4 u;
    u.x = bf16_rne(lo.x) | (uint32_t(bf16_rne(lo.y)) << 16);
    u.y = bf16_rne(lo.z) | (uint32_t(bf16_rne(lo.w)) << 16);
    u.z = bf16_rne(hi.x) | (uint32_t(bf16_rne(hi.y)) << 16);
    u.w = bf16_rne(hi.z) | (uint32_t(bf16_rne(hi.w)) << 16);
    return bits_to_bf16x8(u);
  } else {
    const bf16_t* p = static_cast<const bf16_t*>(x) + (int64_t)row * K + k;
    return bits_to_bf16x8(*reinterpret_cast<const uint4*>(p));
  }
}

struct ProjArgs {
  const void* x;          // [rows][K]: bf16 (QKV) or f32 (output projection)
  const uint4* w;         // packed weight, N columns
  int rows, K, N;
  // QKV: columns [0, nq) -> q, [nq, nq + nkv) -> k, the rest -> v (bf16 [rows][n])
  int nq, nkv;
  bf16_t *q, *k, *v;
  // output projection: h [rows][N] f32 += bf16(y); x_next = bf16(h)
  float* h;
  bf16_t* x_next;
  // QKV with UpdateKV (rows = batch * W1 window rows): row W1-1 of every
  // sequence goes to k / v ([batch][nkv]), the n_upd rows before it overwrite the
  // sequence's last n_upd stored tokens, whose pages' digests are recomputed
  int W1, n_upd, P, D, hk, max_pages, num_phys;
  bf16_t *kc, *vc, *dg;
  const int32_t* pt;
  const int32_t* seq_lens;
};

constexpr int PJ_MAX_BATCH = 16 * PJ_MAX_ROW_TILES;

template <int MT, bool OUT, int U, bool UPD = false, int CT = 1, int NW = PJ_WAVES>
__global__ void __launch_bounds__(64 * NW) proj_kernel(ProjArgs a) {
  __shared__ float red[NW][4][64];
  __shared__ int s_len[UPD ? PJ_MAX_BATCH : 1];
  __shared__ uint16_t s_val[UPD ? CT : 1][UPD ? MT * 16 : 1][16];
  if constexpr (UPD) {
    // sequence lengths before the step's append, loaded under the weight stream
    const int nb = a.rows / a.W1;
    if ((int)threadIdx.x < nb) s_len[threadIdx.x] = a.seq_lens[threadIdx.x];
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int ln16 = lane & 15, g4 = lane >> 4;
  const int tile0 = blockIdx.x * CT;  // CT column tiles share each load of the rows
  const int steps = a.K / 32, per_wave = steps / NW;
  const int s0 = wave * per_wave;
  const uint4* wp = a.w + ((int64_t)tile0 * steps + s0) * 64 + lane;
  f32x4 acc[CT][MT];
#pragma unroll
  for (int c = 0; c < CT; ++c)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[c][mt] = f32x4{0.f, 0.f, 0.f, 0.f};
  // U steps per pass, every load of the pass issued before its MFMAs
  for (int s = 0; s < per_wave; s += U) {
    bf16x8 b[U][CT], av[U][MT];
#pragma unroll
    for (int u = 0; u < U; ++u) {
#pragma unroll
      for (int c = 0; c < CT; ++c) b[u][c] = bits_to_bf16x8(wp[((int64_t)c * steps + s + u) * 64]);
      const int k = (s0 + s + u) * 32 + 8 * g4;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) av[u][mt] = load_a<OUT>(a.x, a.rows, a.K, mt * 16 + ln16, k);
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int c = 0; c < CT; ++c)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
          acc[c][mt] =
              __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[u][mt], b[u][c], acc[c][mt], 0, 0, 0);
  }
  // tile by tile through one LDS buffer: output (i, l) of column tile c and row
  // tile mt is row mt*16 + 4*(l/16) + i, column (tile0 + c)*16 + l%16
#pragma unroll
  for (int pass = 0; pass < CT * MT; ++pass) {
    const int c = pass / MT, mt = pass % MT;
    if (pass > 0) __syncthreads();  // the previous tile's sums are read
#pragma unroll
    for (int i = 0; i < 4; ++i) red[wave][i][lane] = acc[c][mt][i];
    __syncthreads();
    const int o = threadIdx.x;
    if (o >= 256) continue;
    const int i = o >> 6, l = o & 63;
    const int row = mt * 16 + 4 * (l >> 4) + i;
    if (row >= a.rows) continue;
    float sum = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) sum += red[w][i][l];
    const int col = (tile0 + c) * 16 + (l & 15);
    const uint16_t y = bf16_rne(sum);
    if constexpr (OUT) {
      const int64_t e = (int64_t)row * a.N + col;
      const float hv = a.h[e] + __uint_as_float(uint32_t(y) << 16);
      a.h[e] = hv;
      a.x_next[e].bits = bf16_rne(hv);
    } else if constexpr (UPD) {
      s_val[c][row][l & 15] = y;
      if (col < a.nq) {
        a.q[(int64_t)row * a.nq + col].bits = y;
        continue;
      }
      const bool is_k = col < a.nq + a.nkv;
      const int c = is_k ? col - a.nq : col - a.nq - a.nkv;
      const int b = row / a.W1, j = row % a.W1;
      if (j == a.W1 - 1) {  // the step's token: appended by the step itself
        (is_k ? a.k : a.v)[(int64_t)b * a.nkv + c].bits = y;
        continue;
      }
      const int len = s_len[b];
      const int pos = len - (a.W1 - 1) + j;  // row j of the window is token t-W+j
      if (j < a.W1 - 1 - a.n_upd || pos < 0) continue;
      const int lp = pos / a.P, slot = pos % a.P;
      if (lp >= a.max_pages) continue;
      const int phys = a.pt[(int64_t)b * a.max_pages + lp];
      if (phys < 0 || phys >= a.num_phys) continue;
      const int h = c / a.D, e = c % a.D;
      const int64_t ph = (int64_t)phys * a.hk + h;
      if (is_k)
        a.kc[(ph * a.P + slot) * a.D + e].bits = y;
      else
        a.vc[(ph * a.D + e) * a.P + slot].bits = y;
    } else {
      if (col < a.nq)
        a.q[(int64_t)row * a.nq + col].bits = y;
      else if (col < a.nq + a.nkv)
        a.k[(int64_t)row * a.nkv + (col - a.nq)].bits = y;
      else
        a.v[(int64_t)row * a.nkv + (col - a.nq - a.nkv)].bits = y;
    }
  }
  if constexpr (UPD) {
    // digests of the pages the update touched, for this workgroup's 16 key
    // columns: element-wise min / max over every stored key of the page, the
    // updated ones taken from s_val (a min / max cannot be narrowed in place)
    if (a.n_upd == 0) return;
    __syncthreads();
    const int nb = a.rows / a.W1;
    const int span = (a.n_upd + a.P - 1) / a.P + 1;  // pages a run of n_upd can touch
#pragma unroll
    for (int c = 0; c < CT; ++c) {
    const int col0 = (tile0 + c) * 16;
    if (col0 < a.nq || col0 >= a.nq + a.nkv) continue;
    const int c0 = col0 - a.nq, h = c0 / a.D;
    for (int o = threadIdx.x; o < nb * span * 16; o += blockDim.x) {
      const int cl = o & 15, pi = (o >> 4) % span, b = (o >> 4) / span;
      const int e = c0 % a.D + cl;
      const int len = s_len[b];
      const int start = max(len - a.n_upd, 0);
      const int lp = start / a.P + pi;
      if (lp >= a.max_pages || lp * a.P >= len) continue;
      const int phys = a.pt[(int64_t)b * a.max_pages + lp];
      if (phys < 0 || phys >= a.num_phys) continue;
      const int filled = min(a.P, len - lp * a.P);
      const int64_t ph = (int64_t)phys * a.hk + h;
      float lo = 0.f, hi = 0.f;
      for (int sl = 0; sl < filled; ++sl) {
        const int pos = lp * a.P + sl;
        float f;
        if (pos >= start)
          f = to_f32(bf16_t{s_val[c][b * a.W1 + (pos - len + a.W1 - 1)][cl]});
        else
          f = to_f32(a.kc[(ph * a.P + sl) * a.D + e]);
        if (sl == 0) {
          lo = f;
          hi = f;
        } else {
          if (f < lo) lo = f;
          if (hi < f) hi = f;
        }
      }
      bf16_t* drow = a.dg + (((int64_t)b * a.hk + h) * a.max_pages + lp) * 2 * a.D;
      drow[e].bits = static_cast<uint16_t>(__float_as_uint(lo) >> 16);
      drow[a.D + e].bits = static_cast<uint16_t>(__float_as_uint(hi) >> 16);
    }
    }
  }
}

// The most reduction steps per pass whose operands fit the registers: 8 for
// one or two row tiles, 4 for three or four, 2 beyond.
constexpr int max_unroll(int mt) { return mt <= 2 ? 8 : mt <= 4 ? 4 : 2; }

template <int MT, bool OUT, bool UPD>
void launch_proj_mt(const ProjArgs& a, hipStream_t s) {
  // as many reduction steps per pass as the wavefront's share and the registers
  // allow, so that a share takes as few dependent round trips to memory as
  // possible (the share, K / 512 steps, is even)
  // query / key / value with three to five row tiles: two column tiles per
  // workgroup where N allows, halving the re-reads of the rows (every workgroup
  // reads all of them); not for the output projection, whose 4096 columns would
  // then leave half the compute units without a workgroup
  constexpr int UM = max_unroll(MT);
  constexpr int CT = (!OUT && MT >= 3 && MT <= 5) ? 2 : 1;
  const int per_wave = a.K / 32 / PJ_WAVES;
  const dim3 block(64 * PJ_WAVES);
  if (CT == 2 && a.N % 32 == 0) {
    const dim3 grid(a.N / 32);
    constexpr int UC = MT >= 4 ? 2 : UM;  // four or five row tiles: 4 steps would spill
    if (per_wave % UC == 0)
      proj_kernel<MT, OUT, UC, UPD, CT><<<grid, block, 0, s>>>(a);
    else
      proj_kernel<MT, OUT, 2, UPD, CT><<<grid, block, 0, s>>>(a);
    return;
  }
  const dim3 grid(a.N / 16);
  if constexpr (MT == 1) {
    if ((int)grid.x > compute_units() && (a.K / 32 / 8) % 8 == 0) {
      // one row tile and more column tiles than compute units: eight wavefronts
      // per workgroup (two passes of eight steps), so that every workgroup of
      // the launch is resident at once instead of a second, half-empty round
      proj_kernel<MT, OUT, 8, UPD, 1, 8><<<grid, dim3(64 * 8), 0, s>>>(a);
      return;
    }
  }
  if (per_wave % UM == 0)
    proj_kernel<MT, OUT, UM, UPD><<<grid, block, 0, s>>>(a);
  else if (UM > 4 && per_wave % 4 == 0)
    proj_kernel<MT, OUT, (UM > 4 ? 4 : 2), UPD><<<grid, block, 0, s>>>(a);
  else
    proj_kernel<MT, OUT, 2, UPD><<<grid, block, 0, s>>>(a);
}

template <bool OUT, bool UPD>
hipError_t launch_proj(const ProjArgs& a, hipStream_t s) {
  switch ((a.rows + 15) / 16) {
    case 1: launch_proj_mt<1, OUT, UPD>(a, s); break;
    case 2: launch_proj_mt<2, OUT, UPD>(a, s); break;
    case 3: launch_proj_mt<3, OUT, UPD>(a, s); break;
    case 4: launch_proj_mt<4, OUT, UPD>(a, s); break;
    case 5: launch_proj_mt<5, OUT, UPD>(a, s); break;
    case 6: launch_proj_mt<6, OUT, UPD>(a, s); break;
    default: launch_proj_mt<7, OUT, UPD>(a, s); break;
  }
  return hipGetLastError();
}

// [K][N] row-major -> packed tiles; one thread per 8-element group.
__global__ void pack_kernel(const bf16_t* __restrict__ w, int K, int N, uint4* __restrict__ out) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t total = (int64_t)K * N / 8;
  if (idx >= total) return;
  const int lane = (int)(idx & 63);
  const int64_t ts = idx >> 6;           // tile * steps + step
  const int steps = K / 32;
  const int tile = (int)(ts / steps), step = (int)(ts % steps);
  const int col = tile * 16 + (lane & 15);
  const int k0 = step * 32 + 8 * (lane >> 4);
  uint32_t h[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) h[j] = w[(int64_t)(k0 + j) * N + col].bits;
  out[idx] = make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16),
                        h[6] | (h[7] << 16));
}

retro_status status_of(hipError_t e) { return e == hipSuccess ? RETRO_OK : RETRO_EHIP; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool proj_shape_ok(int rows, int K, int N) {
  return rows >= 1 && rows <= 16 * PJ_MAX_ROW_TILES && K > 0 &&
         K % (32 * PJ_WAVES * PJ_MIN_STEPS) == 0 &&
         N > 0 && N % 16 == 0;
}

}  // namespace

hipError_t launch_project_qkv_update(const Geometry& g, const retro_kv_cache& c, const void* x,
                                     int k, const void* w_packed, int n_upd, void* q,
                                     void* k_new, void* v_new, hipStream_t s) {
  ProjArgs a{};
  a.x = x;
  a.w = static_cast<const uint4*>(w_packed);
  a.W1 = g.W + 1;
  a.rows = g.batch * a.W1;
  a.K = k;
  a.nq = g.hq * g.D;
  a.nkv = g.hk * g.D;
  a.N = a.nq + 2 * a.nkv;
  a.q = static_cast<bf16_t*>(q);
  a.k = static_cast<bf16_t*>(k_new);
  a.v = static_cast<bf16_t*>(v_new);
  a.n_upd = n_upd;
  a.P = g.P;
  a.D = g.D;
  a.hk = g.hk;
  a.max_pages = g.max_pages;
  a.num_phys = g.num_phys;
  a.kc = static_cast<bf16_t*>(c.k_cache);
  a.vc = static_cast<bf16_t*>(c.v_cache);
  a.dg = static_cast<bf16_t*>(c.digest);
  a.pt = c.page_table;
  a.seq_lens = c.seq_lens;
  return launch_proj<false, true>(a, s);
}

bool project_qkv_update_supported(const Geometry& g, int k) {
  return g.dtype == RETRO_BF16 && proj_shape_ok(g.batch * (g.W + 1), k, (g.hq + 2 * g.hk) * g.D) &&
         g.batch <= PJ_MAX_BATCH && g.D % 16 == 0;
}

}  // namespace retro

namespace {

// fp32 projections (fp32 stacks): one thread per output element (row r =
// blockIdx.y, column j), an in-order fused multiply-add chain over the k inputs;
// the row's inputs staged through LDS 1024 at a time, the weight read by
// consecutive columns (coalesced).
constexpr int kF32Threads = 256;
constexpr int kF32Chunk = 1024;
__global__ void __launch_bounds__(kF32Threads) project_f32_kernel(const float* __restrict__ x,
                                                                  int K, const float* __restrict__ w,
                                                                  int N, float* __restrict__ y,
                                                                  int accumulate) {
  __shared__ float xs[kF32Chunk];
  const int r = blockIdx.y;
  const int j = blockIdx.x * kF32Threads + threadIdx.x;
  const float* xr = x + (int64_t)r * K;
  float acc = 0.f;
  for (int i0 = 0; i0 < K; i0 += kF32Chunk) {
    const int cnt = min(kF32Chunk, K - i0);
    __syncthreads();
    for (int i = threadIdx.x; i < cnt; i += kF32Threads) xs[i] = xr[i0 + i];
    __syncthreads();
    if (j < N) {
      const float* wc = w + (int64_t)i0 * N + j;
      for (int i = 0; i < cnt; ++i) acc = fmaf(xs[i], wc[(int64_t)i * N], acc);
    }
  }
  if (j < N) {
    float* yo = y + (int64_t)r * N + j;
    *yo = accumulate ? *yo + acc : acc;
  }
}

}  // namespace

extern "C" {

retro_status retro_pack_weight(const void* w, int32_t k, int32_t n, void* w_packed,
                               void* stream) {
  if (!w || !w_packed || k <= 0 || n <= 0) return RETRO_EINVAL;
  if (!retro::aligned16(w_packed)) return RETRO_EINVAL;
  if (k % 32 != 0 || n % 16 != 0) return RETRO_EUNSUPPORTED;
  const int64_t groups = (int64_t)k * n / 8;
  const int threads = 256;
  const int64_t blocks = (groups + threads - 1) / threads;
  if (blocks > 0x7fffffff) return RETRO_EUNSUPPORTED;
  retro::pack_kernel<<<(unsigned)blocks, threads, 0, (hipStream_t)stream>>>(
      static_cast<const retro::bf16_t*>(w), k, n, static_cast<uint4*>(w_packed));
  return retro::status_of(hipGetLastError());
}

retro_status retro_project_qkv(const void* x, int32_t rows, int32_t k, const void* w_packed,
                               int32_t n_q, int32_t n_kv, void* q, void* k_out, void* v,
                               void* stream) {
  if (!x || !w_packed || !q || !k_out || !v || rows < 0 || k <= 0 || n_q <= 0 || n_kv <= 0)
    return RETRO_EINVAL;
  if (rows == 0) return RETRO_OK;
  if (!retro::aligned16(x) || !retro::aligned16(w_packed)) return RETRO_EINVAL;
  const int n = n_q + 2 * n_kv;
  if (!retro::proj_shape_ok(rows, k, n) || n_q % 16 != 0 || n_kv % 16 != 0)
    return RETRO_EUNSUPPORTED;
  retro::ProjArgs a{};
  a.x = x;
  a.w = static_cast<const uint4*>(w_packed);
  a.rows = rows;
  a.K = k;
  a.N = n;
  a.nq = n_q;
  a.nkv = n_kv;
  a.q = static_cast<retro::bf16_t*>(q);
  a.k = static_cast<retro::bf16_t*>(k_out);
  a.v = static_cast<retro::bf16_t*>(v);
  return retro::status_of(retro::launch_proj<false, false>(a, (hipStream_t)stream));
}

retro_status retro_project_out(const float* o, int32_t rows, int32_t k, const void* w_packed,
                               int32_t n, float* h, void* x_next, void* stream) {
  if (!o || !w_packed || !h || !x_next || rows < 0 || k <= 0 || n <= 0) return RETRO_EINVAL;
  if (rows == 0) return RETRO_OK;
  if (!retro::aligned16(o) || !retro::aligned16(w_packed)) return RETRO_EINVAL;
  if (!retro::proj_shape_ok(rows, k, n)) return RETRO_EUNSUPPORTED;
  retro::ProjArgs a{};
  a.x = o;
  a.w = static_cast<const uint4*>(w_packed);
  a.rows = rows;
  a.K = k;
  a.N = n;
  a.h = h;
  a.x_next = static_cast<retro::bf16_t*>(x_next);
  return retro::status_of(retro::launch_proj<true, false>(a, (hipStream_t)stream));
}

retro_status retro_project_f32(const float* x, int32_t rows, int32_t k, const float* w,
                               int32_t n, float* y, int32_t accumulate, void* stream) {
  if (!x || !w || !y || rows < 0 || k <= 0 || n <= 0) return RETRO_EINVAL;
  if (rows == 0) return RETRO_OK;
  if (rows > 65535 || (int64_t)rows * n >= (int64_t(1) << 31)) return RETRO_EUNSUPPORTED;
  const dim3 grid((unsigned)((n + kF32Threads - 1) / kF32Threads), (unsigned)rows);
  project_f32_kernel<<<grid, kF32Threads, 0, (hipStream_t)stream>>>(
      x, k, w, n, y, accumulate ? 1 : 0);
  return retro::status_of(hipGetLastError());
}

}  // extern "C"
