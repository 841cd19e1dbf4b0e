// PageSelect by threshold (Alg. 1; Sec. 2.1): the k pages of one (sequence, KV
// head) with the highest scores, ties going to the lower page index, found as
// the k-th largest score and the number of pages tying with it that are kept.
//
// The first NTS threads of the workgroup hold PER pages of the head each, page
// p = j * NTS + tid for stripe j, as order-preserving 32-bit keys (the other
// threads hold none but take part in the barriers).  The k-th largest key T is
// found by radix rounds over rel = key - min(key): a round histograms the next
// 12 bits of the keys that still match T's digits so far into 4096 fine bins
// (LDS atomics, few of which meet on one bin), the wavefronts sum them into 64
// coarse bins of 64, and then every wavefront locates T's bin by itself,
// scanning the coarse bins from the top and then the 64 fine bins of the
// coarse bin it lands in (two LDS reads and two wavefront prefix sums), so a
// round costs two barriers.  The rounds stop as soon
// as T's bin holds exactly the keys still to be taken, or the digits reach bit 0
// (the bin then holds keys equal to T).  A page is kept if its key's digits so
// far are above T's, or equal to them and fewer than `need` such pages have a
// lower index.  Its rank among the kept pages in page order is found with
// ballots: per (stripe, wavefront) counts go to LDS and one prefix sum over
// that table, in page order, gives every kept page its output slot.
#pragma once

#include "roles.h"

namespace retro {

constexpr int kThrBits = 12;
constexpr int kThrBins = 1 << kThrBits;    // fine bins of a round
constexpr int kThrCoarse = kThrBins / 64;  // coarse bins, 64 fine bins each

// LDS of the selection.  fine: two rounds' histograms, zero on entry (the
// caller clears them and passes a barrier before the call); coarse: their
// sums, written by each round.
template <int PER, int NW>
struct ThrLds {
  uint32_t fine[2][kThrBins];
  uint32_t coarse[2][kThrCoarse];
  uint32_t mn[NW], mx[NW];
  int cnt_gt[PER * NW], cnt_eq[PER * NW];
};

// Zeroes the histograms (every thread of the workgroup takes part; a barrier
// must follow before threshold_select).
template <int PER, int NW>
__device__ __forceinline__ void thr_clear(ThrLds<PER, NW>& L) {
  uint32_t* f = &L.fine[0][0];
  for (int i = thread_index(); i < 2 * kThrBins; i += NW * 64) f[i] = 0u;
}

// The kept pages of one head.  key[j]: order key of page j * NTS + tid (for
// tid < NTS <= 64 * NW, the workgroup's NW wavefronts), meaningful for pages
// < n; k: pages to keep (k >= n keeps every page).  kmin / kmax: the smallest
// and largest key of the pages < n, when known already (MINMAX false; then
// needed in the wavefronts that hold stripes only: the others take them from
// wavefront 0 through LDS after the first barrier), else computed here.  On return pos[j] is the page's slot among the kept pages in
// page order, -1 if it is not kept (or >= n, or tid >= NTS).  All threads of
// the workgroup call it (it contains barriers).
template <int PER, int NW, int NTS, bool MINMAX = true>
__device__ __forceinline__ void threshold_select(ThrLds<PER, NW>& L, const uint32_t (&key)[PER],
                                                 int n, int k, int (&pos)[PER],
                                                 uint32_t kmin_in = 0u, uint32_t kmax_in = 0u) {
  static_assert(NTS % 64 == 0 && NTS <= 64 * NW && kThrCoarse % NW == 0, "selection shape");
  constexpr int NE = PER * NW;             // (stripe, wavefront) table entries
  constexpr int NCH = (NE + 63) / 64;
  constexpr int CPW = kThrCoarse / NW;     // coarse bins summed by each wavefront
  constexpr int LPC = 64 / CPW;            // lanes per coarse bin
  constexpr int FPL = 64 / LPC;            // fine bins per lane
  const int tid = thread_index(), lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  auto valid = [&](int j) { return tid < NTS && j * NTS + tid < n; };
  const bool all = k >= n;
  const bool none = k <= 0;

  uint32_t kmin = 0u;
  uint64_t prefix = 0u;  // T's digits of rel, bits [lo, 32)
  int lo = 32;
  int need = k;          // keys still to take among those matching the prefix
  if (!all && !none) {   // uniform
    uint32_t a = kmin_in, b = kmax_in;
    if constexpr (MINMAX) {
      a = 0xFFFFFFFFu;
      b = 0u;
#pragma unroll
      for (int j = 0; j < PER; ++j)
        if (valid(j)) {
          a = min(a, key[j]);
          b = max(b, key[j]);
        }
      a = wave_umin(a);
      b = wave_umax(b);
      if (lane == 0) {
        L.mn[w] = a;
        L.mx[w] = b;
      }
      __syncthreads();
      a = 0xFFFFFFFFu;
      b = 0u;
#pragma unroll
      for (int i = 0; i < NW; ++i) {
        a = min(a, L.mn[i]);
        b = max(b, L.mx[i]);
      }
    }
    if constexpr (!MINMAX) {
      if (tid == 0) {
        L.mn[0] = a;
        L.mx[0] = b;
      }
    }
    kmin = a;
    const uint32_t range = b - a;
    int hi = range ? 32 - __clz((int)range) : 1;
    lo = hi;
    prefix = 0u;
#pragma unroll 1
    for (int round = 0;; ++round) {
      lo = max(hi - kThrBits, 0);
      const int buf = round & 1;
      if (round == 2) {
        // a third round (keys spread over more than 24 bits) reuses the first
        // round's histograms: every wavefront finished scanning them before
        // the second round's barriers
        uint32_t* f = &L.fine[0][0];
        for (int i = tid; i < kThrBins; i += 64 * NW) f[i] = 0u;
        __syncthreads();
      }
      const uint32_t dmask = (1u << (hi - lo)) - 1u;
#pragma unroll
      for (int j = 0; j < PER; ++j) {
        const uint64_t rel = (uint64_t)(key[j] - kmin);
        if (valid(j) && (rel >> hi) == prefix) {
          atomicAdd(&L.fine[buf][(uint32_t)(rel >> lo) & dmask], 1u);
        }
      }
      __syncthreads();
      if constexpr (!MINMAX) {
        if (round == 0 && tid >= NTS) {  // wavefront-uniform: no stripes, no key range
          kmin = L.mn[0];
          const uint32_t r0 = L.mx[0] - kmin;
          hi = r0 ? 32 - __clz((int)r0) : 1;
          lo = max(hi - kThrBits, 0);
        }
      }
      {  // coarse bin w * CPW + lane / LPC = the sum of its 64 fine bins
        const int cbin = w * CPW + lane / LPC;
        const uint32_t* f = &L.fine[buf][cbin * 64 + (lane % LPC) * FPL];
        uint32_t x = 0u;
#pragma unroll
        for (int i = 0; i < FPL; i += 4) {
          const uint4 q4 = *reinterpret_cast<const uint4*>(f + i);
          x += q4.x + q4.y + q4.z + q4.w;
        }
#pragma unroll
        for (int m = 1; m < LPC; m *= 2) x += (uint32_t)__shfl_xor((int)x, m);
        if (lane % LPC == 0) L.coarse[buf][cbin] = x;
      }
      __syncthreads();
      // T's coarse bin: bins from the top, lane l holding coarse bin 63 - l
      const int cx = (int)L.coarse[buf][kThrCoarse - 1 - lane];
      const int ci = wave_inclusive_scan(cx);
      const int lc = __builtin_ctzll(wave_ballot(ci >= need));
      const int above_c = __builtin_amdgcn_readlane(ci - cx, lc);
      const int cb = kThrCoarse - 1 - lc;
      // T's fine bin within it
      const int fx = (int)L.fine[buf][cb * 64 + 63 - lane];
      const int fi = wave_inclusive_scan(fx) + above_c;
      const int lf = __builtin_ctzll(wave_ballot(fi >= need));
      const int above = __builtin_amdgcn_readlane(fi - fx, lf);
      const int inbin = __builtin_amdgcn_readlane(fx, lf);
      need -= above;
      prefix = (prefix << (hi - lo)) | (uint64_t)(cb * 64 + 63 - lf);
      hi = lo;
      if (inbin == need || lo == 0) break;  // uniform: every wavefront computed the same
    }
  }

  // Compaction in page order.  gt: the key's digits are above T's; eq: equal
  // to them (then kept if fewer than `need` eq pages have a lower index).
  uint64_t bg[PER], be[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const uint64_t km = (uint64_t)(key[j] - kmin) >> lo;
    const bool v = valid(j) && !none;
    const bool gt = v && (all || km > prefix);
    const bool eq = v && !all && km == prefix;
    bg[j] = wave_ballot(gt);
    be[j] = wave_ballot(eq);
    if (lane == 0) {
      L.cnt_gt[j * NW + w] = __popcll(bg[j]);
      L.cnt_eq[j * NW + w] = __popcll(be[j]);
    }
  }
  __syncthreads();
  int sg[NCH], se[NCH];  // exclusive prefix sums of the tables, entry c * 64 + lane
  int cg = 0, ce = 0;
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const int e = c * 64 + lane;
    const int vg = e < NE ? L.cnt_gt[e] : 0;
    const int ve = e < NE ? L.cnt_eq[e] : 0;
    const int ig = wave_inclusive_scan(vg) + cg;
    const int ie = wave_inclusive_scan(ve) + ce;
    sg[c] = ig - vg;
    se[c] = ie - ve;
    cg = __builtin_amdgcn_readlane(ig, 63);
    ce = __builtin_amdgcn_readlane(ie, 63);
  }
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int e = j * NW + w;  // wavefront-uniform
    int bgl = 0, bel = 0;
#pragma unroll
    for (int c = 0; c < NCH; ++c)
      if (e / 64 == c) {
        bgl = __builtin_amdgcn_readlane(sg[c], e % 64);
        bel = __builtin_amdgcn_readlane(se[c], e % 64);
      }
    const bool is_gt = (bg[j] >> lane) & 1u;
    const bool is_eq = (be[j] >> lane) & 1u;
    const int gb = bgl + lanes_below(bg[j]);
    const int eb = bel + lanes_below(be[j]);
    int p = -1;
    if (is_gt) p = gb + min(eb, need);
    if (is_eq && eb < need) p = gb + eb;
    pos[j] = p;
  }
}

}  // namespace retro
