// A whole decode step in a single launch, for shapes whose workgroups all fit
// on the GPU at once (the Llama-class layers): Alg. 1's AppendKV, PageSelect,
// attention, MergeOutput and CacheOutput, Alg. 2, eq. (quest_score),
// eq. (update-org), eq. (update-sup) and eq. (merged_attn_general).
//
// Each KV head (sequence b, head h) gets NW workgroups; workgroup j of the head
//   1. scores the head's pages [j * ppb, (j + 1) * ppb), appending the step's
//      token where its page is among them (score_role);
//   2. publishes every score as one 64-bit word: the score's bits and the
//      launch's epoch (tag), and the smallest and largest key of its share in
//      two more, written device-coherently by one wavefront;
//   3. loads the head's score words, each thread of the other wavefronts its
//      stripe of pages, until every word of a page of the sequence carries
//      this launch's epoch (the data are their own signal: no counter, no
//      barrier across workgroups);
//   4. computes the head's selection by threshold (threshold.h) and writes the
//      page list of its split of the kept pages into LDS; the head's writer
//      workgroup (j = 0) also keeps the whole selection there;
//   5. runs the attention of its split (attend_role) and writes the split's
//      partial output rows device-coherently; once a wavefront's rows are
//      written through, it publishes their log-normalisers as tagged words;
//   6. the head's writer workgroup stores the selection rows, mask values,
//      count and Alg. 2's last_loaded update (after every workgroup of the
//      head has read last_loaded: their score words say so) and a tagged
//      head word (selection done);
//   7. combine + merge units, spread over the head's workgroups, wait for the
//      log-normaliser words of their rows in every split, then read the
//      partial rows and merge them into the output cache (merge_unit);
//   8. one wavefront per sequence advances seq_lens once every head of the
//      sequence has published its head word (every reader of seq_lens in
//      the launch has then read it).
//
// Epoch.  Every workgroup has a line of its own in the workspace holding the
// epoch of the last launch it ran (and a fingerprint of the geometry); it reads
// the line at its start and its publisher wavefront stores the next epoch.  All
// workgroups of a launch run once per launch, so the lines agree, and the
// epoch is the same in every workgroup of the launch.  Epochs count 1, 2, ...,
// 2^31 - 1, then 1 again: 31 bits, because the log-normaliser and head words
// keep their top bit for a failure flag, and never 0, the tag of a word no
// launch has written.  A word written by an earlier launch carries another
// epoch unless exactly a multiple of 2^31 - 1 launches on this workspace have
// passed without rewriting it.  A workspace last used with another geometry is
// refused by the fingerprint: the sticky error word is set and no wait is
// entered.
//
// Coherence (without fences, which would write back or invalidate whole L2s):
//   - a score word is written with one device-coherent (sc1) 64-bit store and
//     read with device-coherent loads, which are not served from a
//     non-coherent L2 copy: a reader sees either an older word (an older tag)
//     or this launch's word, never a torn one;
//   - the step's token key and value are stored into the cache by the
//     workgroup whose share holds the token's page, with plain stores and no
//     wait: they are for later launches.  In this launch the gather of the
//     token's page takes the token's key row and value column from the step's
//     input (k_new, v_new) into LDS, over whatever the cache slot holds; the
//     page's other tokens were stored by earlier launches;
//   - the gather uses plain loads of lines that no workgroup of this launch
//     writes, apart from the token's bytes (replaced as above); no L2 holds a
//     line from before the launch (the launch's acquire at its start), so no
//     stale copy can be hit;
//   - the partial output rows go out as device-coherent 16-byte stores; each
//     wavefront waits until they are acknowledged (s_waitcnt 0) before it
//     stores its tagged log-normaliser words, and the combine reads the rows
//     with device-coherent loads only after it has seen those tags;
//   - the writer's plain stores (selection rows, mask, count, last_loaded) and
//     the seq_lens advance are read by later launches only, except
//     last_loaded and seq_lens, which every workgroup reads at its start: the
//     writer stores last_loaded only after seeing every score word of its head
//     (each issued after the issuing workgroup's loads had returned), and
//     seq_lens advances only after every head word of the sequence;
//   - each output-cache slot is read and written by one merge unit only.
//
// Waits are bounded: past spin_limit polls the sticky error word is set and the
// workgroup goes on with what it has; the combine then writes NaN outputs and
// leaves the output cache, last_loaded and seq_lens as they were.
#include "threshold.h"

namespace retro {
namespace {

constexpr int kThreads = 512;
constexpr uint64_t kEpochs = 0x7FFFFFFFull;  // epochs 1 .. 2^31 - 1
constexpr int kWaves = kThreads / 64;

struct StepAttendArgs {
  AttendArgs a;
  float* scores;       // [batch * h_k][max_pages] fp32: every score, for retro_copy_scores
  int32_t* A;          // last_loaded: read for the mask values, updated after the step
  int32_t* tok_out;    // [batch * h_k]: the step token's page if it is not kept, else -1
  int32_t* err;        // sticky error word
  const void* k_new;   // the step's token, [batch][h_k][d] (null: no token)
  const void* v_new;
  int spin_limit;      // polls before a wait gives up
  uint32_t tag_bias;   // added to the awaited tag (tests: makes every wait give up)
  // the combine + merge in the same launch (m.o_out null: partials only)
  MergeArgs m;
  uint64_t* lse_tag;   // [batch * h_k][R][splits]: tagged log-normaliser of each partial row
  uint64_t* head_tag;  // [batch * h_k]: tagged once the head's first workgroup has selected
};

template <typename T, int D, int PER, int SITERS>
struct StepLds {
  union {
    T stage[2 * Tiles<T, D>::BUF_ELEMS];
    ThrLds<PER, kWaves> thr;
  } u;
  float sq[2 * 16 * D];           // the group's current queries (fp32, q+ then q-) while scoring
  float share[SITERS * kWaves * 4];  // this workgroup's scores
  T dig[2 * D];                   // the token page's widened digest row
  int s_phys[kMaxSplitPages], s_len[kMaxSplitPages], s_mask[kMaxSplitPages];
  // the head writer's selection (page, mask value per kept slot) and the
  // token's page if it is not kept (-1 otherwise), stored after the attention
  int wsel[PER * (kThreads - 64)], wmsk[PER * (kThreads - 64)];  // up to the largest page count
  int wtok;
  int s_tok;
  uint32_t epoch, fp_seen;
  int bad;                        // this workgroup failed (see StepAttendArgs::err)
  int k;
};

// Wavefront 7 issues every store of the score phase (the score words, the
// share's key range, the plain scores, the token's key and value, the digest
// row of its page) and counts the workgroup in; wavefronts 0-6 hold the
// selection's stripes and poll.  On this GPU a wavefront's loads and stores
// retire in order: a poll issued behind device-coherent stores would wait for
// their write-through.
constexpr int kPollThreads = kThreads - 64;

// The kernel's parameters in order: the layout of its kernel-argument segment.
template <typename T>
struct StepParams {
  T* dg;
  uint32_t mp, ppb, nw, ngrid;
  const T* q_cur;
  uint32_t hk, q_bstride;
  uint32_t* ctl;
  uint64_t* tagged;
  uint32_t fingerprint;
  StepAttendArgs sa;
};

// Leading arguments (the pointers and sizes the first loads need: queries and
// digests) come before the argument block so that they can be preloaded into
// scalar registers: those loads then go out without waiting for the
// kernel-argument segment.  The argument block itself is read through the
// segment pointer, passed through an empty asm statement once those loads are
// out (tok_of): the compiler would otherwise load its fields (and wait for
// them, several scalar round trips) ahead of the first vector loads.
template <typename T, int D, int PER, int SITERS, int GC>
__global__ void __launch_bounds__(kThreads) step_attend_kernel(
    T* __restrict__ dg, uint32_t mp, uint32_t ppb, uint32_t nw, uint32_t ngrid,
    const T* __restrict__ q_cur, uint32_t hk, uint32_t q_bstride, uint32_t* __restrict__ ctl,
    uint64_t* __restrict__ tagged, uint32_t fingerprint, StepAttendArgs sa_param) {
  __shared__ __attribute__((aligned(16))) StepLds<T, D, PER, SITERS> L;
  auto kseg = __builtin_amdgcn_kernarg_segment_ptr();
  const StepAttendArgs* sap = nullptr;  // set by tok_of
  const int tid = thread_index();
  // the wavefront index as a uniform (scalar) value: indices and offsets
  // derived from it (the merge units' rows) stay in scalar registers
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const uint32_t u = (uint32_t)xcd_remap(blockIdx.x, ngrid);
  const uint32_t bh = u / nw;
  const uint32_t j = u - bh * nw;
  const int page0 = (int)(j * ppb);
  const int page_end = min(page0 + (int)ppb, (int)mp);
  const int b = (int)(bh / hk), h = (int)bh - b * (int)hk;
  const int gsize = GC > 0 ? GC : sa_param.a.g.G;
  const bool publisher = wave == kWaves - 1;

  // this workgroup's own line: [0, 1] its last epoch (64 bits), [2] the geometry
  // fingerprint, [3] the failure mark (set in every line when a wait of any
  // workgroup gives up); read once the score phase's first loads are out
  // (only failing workgroups write other workgroups' lines)
  uint32_t* line = ctl + ((size_t)bh * nw + j) * 32;
  uint64_t launches = 0;
  uint32_t fp_seen = 0, marked = 0;
  int seq_len = 0, tok_lp = -1;
  StepToken<T> tok{-1, 0, nullptr, nullptr, nullptr, nullptr};
  T tok_kv[2][(D + 63) / 64];  // the publisher's lanes: the token's key and value elements
  T tok_mine[2];               // threads below d: the token's key and value element
  int32_t a_old[PER], phys[PER];
  uint64_t* trow = tagged + (size_t)bh * (mp + 2 * nw);
  uint64_t* hrow = trow + mp;  // per workgroup: the key range of its share

  // ---- 1: this workgroup's share of the head's scores, into LDS
  score_role<T, D, SITERS, true, GC, kThreads>(
      sa_param.a.g, page0, page_end,
      q_cur + (size_t)b * q_bstride + (size_t)h * gsize * D, dg + (size_t)bh * mp * 2 * D, L.sq,
      [&](int& np) {
        asm volatile("" : "+s"(kseg) : : "memory");
        sap = (const StepAttendArgs*)((const __attribute__((address_space(4))) char*)kseg +
                                      offsetof(StepParams<T>, sa));
        const StepAttendArgs& sa = *sap;
        const Geometry& g = sa.a.g;
        // Scalar loads (counted apart from the vector loads in flight, so
        // that their waits do not wait for the digests): the control line,
        // the sequence length and then the token's page-table entry.  No
        // workgroup of the launch writes them before these reads: the line
        // is written by its own workgroup afterwards (or by a failing one),
        // seq_lens only once every workgroup of the sequence has read it.
        const uint32_t cl0 = sload(line), cl1 = sload(line + 1);
        fp_seen = sload(line + 2);
        marked = sload(line + 3);
        launches = (uint64_t)cl1 << 32 | cl0;
        const int pos = sload(sa.a.seq_lens + b);
        // the selection's stripe of last_loaded and page-table entries, with
        // the digests (no load here depends on another)
        const int32_t* arow = sa.A + (size_t)bh * mp;
        const int32_t* prow = sa.a.pt + (size_t)b * mp;
#pragma unroll
        for (int jj = 0; jj < PER; ++jj) {
          const int idx = min(jj * kPollThreads + tid, (int)mp - 1);
          a_old[jj] = arow[idx];
          phys[jj] = prow[idx];
        }
        seq_len = pos;
        if (g.token_pending) {
          const int lp = pos / g.P;
          int ph = (pos >= 0 && lp < (int)mp) ? sload(prow + lp) : -1;
          if (ph >= g.num_phys) ph = -1;
          if (ph >= 0) {
            seq_len = pos + 1;
            tok = make_step_token<T>(g, b, h, pos, ph, sa.k_new, sa.v_new,
                                     const_cast<void*>(sa.a.kc), const_cast<void*>(sa.a.vc));
          }
        }
        np = min((seq_len + g.P - 1) / g.P, (int)mp);
        tok_lp = tok.lp;
        if (tok.lp >= 0) {
          tok_mine[0] = tok.k[min(tid, D - 1)];
          tok_mine[1] = tok.v[min(tid, D - 1)];
        }
        if (publisher && tok.lp >= page0 && tok.lp < page_end) {
#pragma unroll
          for (int r = 0; r < (D + 63) / 64; ++r) {
            const int d = min(lane + 64 * r, D - 1);
            tok_kv[0][r] = tok.k[d];
            tok_kv[1][r] = tok.v[d];
          }
        }
        return tok;
      },
      [&] {
        thr_clear(L.u.thr);
        if (tid == 0) {
          const bool foreign = fp_seen != 0 && fp_seen != fingerprint;
          if (foreign) __hip_atomic_store(sap->err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          L.epoch = (uint32_t)(launches % kEpochs) + 1u;
          L.fp_seen = fp_seen;
          L.bad = foreign || marked != 0;
        }
      },
      [&](int page, float v) { L.share[page - page0] = v; }, L.dig);

  const StepAttendArgs& sa = *sap;
  const Geometry& g = sa.a.g;
  float* srow = sa.scores + (size_t)bh * mp;
  // a wait gave up (wavefront-uniform call): the sticky error word for the
  // caller, and the failure mark in every workgroup's line, so that every later
  // launch on this workspace fails from its start without a shared read
  auto give_up = [&] {
    if (lane == 0) __hip_atomic_store(sa.err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    for (uint32_t i = (uint32_t)lane; i < ngrid; i += 64)
      __hip_atomic_store(ctl + (size_t)i * 32 + 3, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  };
  const int n = min((seq_len + g.P - 1) / g.P, (int)mp);
  // Every load of caller state this workgroup makes (seq_lens, last_loaded, the
  // page table) has returned before its first tagged store below: a workgroup
  // that sees one of its tags may overwrite that state.
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();  // the share's scores and the token page's digest row are in LDS

  // ---- 2: the publisher stores: score words and the share's key range
  // (tagged with the epoch), plain scores for later launches, the token and its
  // page's digest row (for later launches: this launch's gather takes the
  // token from the step's input)
  if (publisher) {
    const uint64_t tag = (uint64_t)L.epoch << 32;
    uint32_t kmn = 0xFFFFFFFFu, kmx = 0u;
    for (int p = page0 + lane; p < min(page_end, n); p += 64) {
      const float v = L.share[p - page0];
      __hip_atomic_store(trow + p, tag | __float_as_uint(v), __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
      srow[p] = v;
      kmn = min(kmn, order_key(v));
      kmx = max(kmx, order_key(v));
    }
    kmn = wave_umin(kmn);
    kmx = wave_umax(kmx);
    if (lane < 2)
      __hip_atomic_store(hrow + 2 * j + lane, tag | (lane == 0 ? kmn : kmx), __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    if (tok.lp >= page0 && tok.lp < page_end) {  // uniform
      constexpr int WORDS = 2 * D * (int)sizeof(T) / 4;
      const uint32_t* src = reinterpret_cast<const uint32_t*>(L.dig);
      uint32_t* dst = reinterpret_cast<uint32_t*>(dg + ((size_t)bh * mp + tok.lp) * 2 * D);
      for (int i = lane; i < WORDS; i += 64) dst[i] = src[i];
#pragma unroll
      for (int r = 0; r < (D + 63) / 64; ++r) {
        const int d = lane + 64 * r;
        if (d < D) {
          tok.k_row[d] = tok_kv[0][r];
          tok.v_col[(int64_t)d * g.P] = tok_kv[1][r];
        }
      }
    }
    if (lane == 0) {
      // this launch's epoch, for the next launch (thread 0 read the line)
      __hip_atomic_store(reinterpret_cast<uint64_t*>(line), (uint64_t)L.epoch, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
      if (L.fp_seen == 0)
        __hip_atomic_store(line + 2, fingerprint, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    if (L.fp_seen == 0) {
      // a fresh workspace: the fingerprint also goes into the lines no
      // workgroup of this geometry owns (u + k * ngrid, k >= 1), so that a
      // later launch of any other geometry finds it in its own line
      for (uint32_t i = u + ngrid * (1u + (uint32_t)lane); i < (uint32_t)kCtlLines; i += 64u * ngrid)
        __hip_atomic_store(ctl + (size_t)i * 32 + 2, fingerprint, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
    }
  }

  const int n_splits = g.n_splits;
  const int split = (int)j % n_splits, rg = (int)j / n_splits;
  const int first = split * g.pages_per_split;
  const bool writer = j == 0;

  // ---- 3-4: the head's scores, then its selection, which fills the split's
  // page list (run by attend_role once its query loads are in flight)
  int k = 0;
  auto select = [&] {
    const uint32_t want = L.epoch + sa.tag_bias;
    const bool bad = L.bad != 0;
    // every page of the sequence in a polling thread's stripe that another
    // workgroup scored (this workgroup's own scores are in LDS), and the key
    // ranges of every share (lane l: word l of the head's range words)
    auto polled = [&](int jj) {
      const int p = jj * kPollThreads + tid;
      return tid < kPollThreads && p < n && (p < page0 || p >= page_end);
    };
    constexpr int HW = 2;  // range words per lane (shares of up to 64 workgroups)
    auto hword = [&](int r) { return (int)(lane + 64 * r) < 2 * (int)nw && !publisher; };
    uint64_t e[PER], hv[HW];
#pragma unroll
    for (int jj = 0; jj < PER; ++jj)
      e[jj] = polled(jj) ? __hip_atomic_load(trow + jj * kPollThreads + tid, __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT)
                         : 0ull;
#pragma unroll
    for (int r = 0; r < HW; ++r)
      hv[r] = hword(r) ? __hip_atomic_load(hrow + lane + 64 * r, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT)
                       : 0ull;
    // meanwhile: the split's page list starts out empty
    if (tid < kMaxSplitPages) {
      L.s_phys[tid] = -1;
      L.s_len[tid] = 0;
      L.s_mask[tid] = 0;
    }
    if (tid == 0) L.s_tok = -1;
    for (int it = 0;; ++it) {
      bool stale = false;
#pragma unroll
      for (int jj = 0; jj < PER; ++jj)
        stale = stale || (polled(jj) && (uint32_t)(e[jj] >> 32) != want);
#pragma unroll
      for (int r = 0; r < HW; ++r) stale = stale || (hword(r) && (uint32_t)(hv[r] >> 32) != want);
      if (wave_ballot(stale) == 0 || bad) break;  // wavefront-uniform
      if (it >= sa.spin_limit) {
        give_up();
        if (lane == 0) L.bad = 1;
        break;
      }
      __builtin_amdgcn_s_sleep(2);
#pragma unroll
      for (int jj = 0; jj < PER; ++jj)
        if (polled(jj) && (uint32_t)(e[jj] >> 32) != want)
          e[jj] = __hip_atomic_load(trow + jj * kPollThreads + tid, __ATOMIC_RELAXED,
                                    __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
      for (int r = 0; r < HW; ++r)
        if (hword(r) && (uint32_t)(hv[r] >> 32) != want)
          hv[r] = __hip_atomic_load(hrow + lane + 64 * r, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    // the head's key range: minimum over the even words, maximum over the odd
    uint32_t kmn = 0xFFFFFFFFu, kmx = 0u;
#pragma unroll
    for (int r = 0; r < HW; ++r)
      if (hword(r)) {
        if ((lane & 1) == 0) kmn = min(kmn, (uint32_t)hv[r]);
        else kmx = max(kmx, (uint32_t)hv[r]);
      }
    kmn = wave_umin(kmn);
    kmx = wave_umax(kmx);
    uint32_t key[PER];
#pragma unroll
    for (int jj = 0; jj < PER; ++jj) {
      const int p = jj * kPollThreads + tid;
      const bool own = p >= page0 && p < page_end;
      const float sv = L.share[max(0, min(p - page0, (int)ppb - 1))];
      key[jj] = order_key(own ? sv : __uint_as_float((uint32_t)e[jj]));
    }
    k = min(min(budget_pages(g, seq_len), n), g.k_max);
    int pos[PER];
    // the arguments the page lists need, read once into vector registers
    // before the selection (the compiler would otherwise reload them in every
    // stripe, each reload waiting for the LDS stores before it)
    int step_m1 = sa.a.step - 1, pps = g.pages_per_split, nphys = g.num_phys, psz = g.P;
    asm volatile("" : "+v"(step_m1), "+v"(pps), "+v"(nphys), "+v"(psz));
    threshold_select<PER, kWaves, kPollThreads, false>(L.u.thr, key, n, k, pos, kmn, kmx);

#pragma unroll
    for (int jj = 0; jj < PER; ++jj) {
      const int p = jj * kPollThreads + tid;
      const int q = pos[jj];
      const int m = p == tok_lp ? step_m1 : a_old[jj];  // Alg. 2's current-page rule
      if (q >= first && q < first + pps) {
        const int ph = (phys[jj] >= 0 && phys[jj] < nphys) ? phys[jj] : -1;
        L.s_phys[q - first] = ph;
        L.s_len[q - first] = ph >= 0 ? min(psz, seq_len - p * psz) : 0;
        L.s_mask[q - first] = m;
        if (p == tok_lp && ph >= 0) L.s_tok = q - first;
      }
      if (writer) {  // into LDS: stores here would hold up the gather's loads behind them
        if (q >= 0) {
          L.wsel[q] = p;
          L.wmsk[q] = m;
        }
        if (tid < kPollThreads && p == tok_lp) L.wtok = q < 0 ? p : -1;
      }
    }
    if (writer && tid == 0 && tok_lp < 0) L.wtok = -1;
    __syncthreads();  // the split's page list is in LDS
  };

  // ---- 5: the split's attention over the window rows; partial outputs
  // written through (sc1), log-normalisers into LDS
  attend_role<T, D, 1, (Tiles<T, D>::PIECES + kThreads - 1) / kThreads, true, true>(
      sa.a, b, h, rg, split, [&] { return seq_len; }, L.u.stage, L.s_phys, L.s_len, L.s_mask,
      &L.s_tok, tok_lp >= 0 ? seq_len - 1 : -1, select,
      PresetList<T>{&k, tok_mine[0], tok_mine[1], sa.m.o_out ? sa.lse_tag : nullptr, &L.epoch,
                    &L.bad});

  // ---- 6: each wavefront has published its rows' log-normalisers (tagged)
  const MergeArgs& m = sa.m;
  // the head writer's selection outputs (rows, mask values, count) and Alg.
  // 2's last_loaded update (with the combine: the whole step), after the
  // attention (stores before it would hold up the gather's loads), by
  // wavefronts 0-3 (the combine's units start on wavefront 0 and wait for the
  // other splits anyway).  Every workgroup of the head has read its stripe of
  // last_loaded before its score tags went out, so the row may change now.
  auto writer_outputs = [&](int t, int nt) {
    int32_t* sel_row = const_cast<int32_t*>(sa.a.sel) + (size_t)bh * g.k_max;
    int32_t* m_row = const_cast<int32_t*>(sa.a.msk) + (size_t)bh * g.k_max;
    int32_t* a_row = sa.A + (size_t)bh * mp;
    const bool upd = m.o_out && L.bad == 0;
    for (int i = t; i < g.k_max; i += nt) {
      const bool kept = i < k;
      const int p = kept ? L.wsel[i] : -1;
      sel_row[i] = p;
      m_row[i] = kept ? L.wmsk[i] : -1;
      if (upd && kept) a_row[p] = sa.a.step;
    }
    if (t == 0) {
      const_cast<int32_t*>(sa.a.nsel)[bh] = k;
      sa.tok_out[bh] = L.wtok;
      if (upd && L.wtok >= 0) a_row[L.wtok] = sa.a.step - 1;
    }
  };
  if (!m.o_out) {  // partials only
    if (writer) writer_outputs(tid, kThreads);
    return;
  }
  const bool failed = L.bad != 0;
  if (publisher && writer && lane == 0) {
    // the head has selected: every workgroup of it has read seq_lens
    const uint64_t hi = (uint64_t)(L.epoch | (failed ? 0x80000000u : 0u)) << 32;
    __hip_atomic_store(sa.head_tag + bh, hi, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }

  // ---- 7: combine + merge (merge_unit): the head's G * max(W, 1) units
  // (window row x of query head gq), spread over its workgroups.  A unit
  // waits until the tags of its rows carry the epoch in every split, then
  // reads the partial rows device-coherently; a failure anywhere in its inputs
  // makes its output rows NaN and leaves its cache slot as it was.
  const uint32_t want = L.epoch + sa.tag_bias;
  auto current = [&](uint64_t w) { return ((uint32_t)(w >> 32) & 0x7FFFFFFFu) == want; };
  auto broken = [&](uint64_t w) { return (w >> 63) != 0; };
  const int xs = g.W > 0 ? g.W : 1;
  const int units = g.G * xs;
  const int nwi = (int)nw;
  // the units in the order x * G + gq (the G two-row units of x = 0 first) to
  // workgroups 1, 2, ..., nw - 1, 0 (the head's writer last), then to the next
  // wavefront; the writer's outputs go out from the wavefronts without units
  // (else the last, after its units)
  const int uw = min(kWaves - 1, (units + nwi - 1) / nwi);
  if (writer && wave >= uw && uw < kWaves - 1) writer_outputs(tid - 64 * uw, kThreads - 64 * uw);
  for (int kk = ((int)j + nwi - 1) % nwi + nwi * wave; kk < units; kk += nwi * kWaves) {  // wavefront-uniform
    const int x = kk / g.G, gq = kk - x * g.G;
    const bool two = g.W > 0 && x == 0;  // rows 0 and W
    const uint64_t* t0 = sa.lse_tag + ((size_t)bh * g.R + x * g.G + gq) * n_splits;
    const uint64_t* t1 = sa.lse_tag + ((size_t)bh * g.R + g.W * g.G + gq) * n_splits;
    const bool l0 = lane < n_splits, l1 = two && lane < n_splits;
    const UnitPos up{x, gq, h, b};  // merge unit (bh * G + gq) * xs + x
    // the unit's output-cache row, loaded while the tags are awaited (merge_unit
    // would load it just ahead of the partial rows, and the compiler waits for
    // it before their loads go out: a second round trip)
    const int64_t ci = unit_cache_row(m, up);
    Row<D> pre{};
    if (ci >= 0) pre = get<D>(m.o_cache, m.l_cache, ci);  // wavefront-uniform
    uint64_t w0 = l0 ? __hip_atomic_load(t0 + lane, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0ull;
    uint64_t w1 = l1 ? __hip_atomic_load(t1 + lane, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0ull;
    bool timed_out = false;
    for (int it = 0;; ++it) {
      const bool stale = (l0 && !current(w0)) || (l1 && !current(w1));
      if (wave_ballot(stale) == 0) break;
      if (it >= sa.spin_limit) {
        timed_out = true;
        give_up();
        break;
      }
      __builtin_amdgcn_s_sleep(2);
      if (l0 && !current(w0)) w0 = __hip_atomic_load(t0 + lane, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (l1 && !current(w1)) w1 = __hip_atomic_load(t1 + lane, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    if (failed || timed_out || wave_ballot((l0 && broken(w0)) || (l1 && broken(w1))) != 0) {
      poison_unit<D>(m, up);
      continue;
    }
    const ZLanes zl{{__uint_as_float((uint32_t)w0), __uint_as_float((uint32_t)w1)}};
    merge_unit<D, 32, true, true, true>(m, up, zl, pre);
  }
  if (writer && uw == kWaves - 1 && wave == kWaves - 1) writer_outputs(lane, 64);

  // ---- 8: seq_lens advances past the token once the first workgroup of every
  // head of the sequence has selected (every workgroup of the sequence has
  // then read seq_lens) and none of them failed
  if (g.token_pending && m.seq_lens && h == 0 && j == 0 && wave == kWaves - 2) {
    const bool lh = lane < (int)hk;
    const uint64_t* ht = sa.head_tag + (size_t)b * hk;
    uint64_t w = lh ? __hip_atomic_load(ht + lane, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0ull;
    bool ok = !failed;
    for (int it = 0; ok; ++it) {
      if (wave_ballot(lh && !current(w)) == 0) break;
      if (it >= sa.spin_limit) {
        ok = false;
        give_up();
        break;
      }
      __builtin_amdgcn_s_sleep(2);
      if (lh && !current(w)) w = __hip_atomic_load(ht + lane, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    if (ok && wave_ballot(lh && broken(w)) == 0 && lane == 0 && tok_lp >= 0) m.seq_lens[b] = seq_len;
  }
}

template <typename T, int D, int PER, int SITERS, int GC>
const void* kernel_ptr() {
  return reinterpret_cast<const void*>(&step_attend_kernel<T, D, PER, SITERS, GC>);
}

// An instantiation's shape: PER pages of the head per polling thread (the
// selection's stripes) and SITERS score passes of 32 pages per workgroup.
template <int PER_, int SITERS_>
struct Shape {
  static constexpr int PER = PER_, SITERS = SITERS_;
};
constexpr int kMaxPer = 10, kMaxSiters = 5;  // the long-context shape

// Score passes a geometry needs: 3 up to 96 pages per workgroup, else 5 (160).
bool long_shape(const Geometry& g) {
  const int nw = g.n_splits * g.n_rgroups;
  const int ppb = (g.max_pages + nw - 1) / nw;
  return g.max_pages > 5 * kPollThreads || ppb > 3 * kWaves * 4;
}

// The instantiation for g: (dtype, d, shape, unrolled group).
template <typename F>
auto dispatch(const Geometry& g, F&& f) {
  const bool g4 = g.G == 4;
  const bool lng = long_shape(g);
  auto per = [&](auto t, auto d) {
    using T = typename decltype(t)::type;
    constexpr int DD = decltype(d)::value;
    auto go = [&](auto shape) {
      using S = decltype(shape);
      return g4 ? f(kernel_ptr<T, DD, S::PER, S::SITERS, 4>(), shape, t, d, std::integral_constant<int, 4>{})
                : f(kernel_ptr<T, DD, S::PER, S::SITERS, 0>(), shape, t, d, std::integral_constant<int, 0>{});
    };
    if (lng) return go(Shape<kMaxPer, kMaxSiters>{});
    if (g.max_pages <= 2 * kPollThreads) return go(Shape<2, 3>{});
    return go(Shape<5, 3>{});
  };
  struct BF { using type = bf16_t; };
  struct F32 { using type = float; };
  if (g.dtype == RETRO_BF16)
    return g.D == 128 ? per(BF{}, std::integral_constant<int, 128>{}) : per(BF{}, std::integral_constant<int, 64>{});
  return g.D == 128 ? per(F32{}, std::integral_constant<int, 128>{}) : per(F32{}, std::integral_constant<int, 64>{});
}

// Workgroups of the kernel that fit on one compute unit at once (cached per
// instantiation and device).
int resident_per_cu(const void* fn) {
  struct Entry { const void* fn; int dev; int n; };
  static Entry cache[64];
  static int used = 0;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  for (int i = 0; i < used; ++i)
    if (cache[i].fn == fn && cache[i].dev == dev) return cache[i].n;
  int n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, fn, kThreads, 0) != hipSuccess) n = 0;
  if (used < 64) cache[used++] = Entry{fn, dev, n};
  return n;
}

uint32_t fingerprint_of(const Geometry& g) {
  // FNV-1a over the shape fields that fix the counter's step (NW) and the
  // score-word layout
  const int32_t f[] = {g.batch, g.hk, g.G, g.D, g.P, g.W, g.max_pages, g.dtype,
                       g.n_splits, g.n_rgroups, g.k_max};
  uint32_t x = 2166136261u;
  for (int32_t v : f)
    for (int i = 0; i < 4; ++i) x = (x ^ ((uint32_t)v >> (8 * i) & 0xFFu)) * 16777619u;
  return x ? x : 1u;
}

}  // namespace

int step_attend_workgroups(const Geometry& g) { return g.n_splits * g.n_rgroups * g.batch * g.hk; }

bool step_attend_supported(const Geometry& g) {
  const int nw = g.n_splits * g.n_rgroups;
  const int ppb = (g.max_pages + nw - 1) / nw;
  if (g.rtw != 1 || g.max_pages > kMaxPer * kPollThreads ||
      ppb > (long_shape(g) ? kMaxSiters : 3) * kWaves * 4 || nw > 64 || g.hk > 64 ||
      g.n_splits > 64)
    return false;
  // partial outputs are read through a buffer resource of 2 GiB
  if ((int64_t)g.batch * g.hk * g.n_splits * g.R * g.D * 4 >= (int64_t(1) << 31)) return false;
  const int grid = step_attend_workgroups(g);
  if (grid > kCtlLines) return false;
  const int per_cu = dispatch(g, [](const void* fn, auto, auto, auto, auto) { return resident_per_cu(fn); });
  return per_cu >= 1 && (int64_t)grid <= (int64_t)per_cu * compute_units();
}

hipError_t launch_step_attend(const Geometry& g, int step, const void* q_window, const void* k_new,
                              const void* v_new, const retro_kv_cache& c,
                              const retro_selection& sel, void* workspace, float* o_ws,
                              float* l_ws, int32_t* tok_out, int32_t* err, int spin_limit,
                              uint32_t tag_bias, const retro_output_cache* oc, float* o_out,
                              float* lse_out, hipStream_t s) {
  if (!step_attend_supported(g) || !tok_out || !err) return hipErrorInvalidValue;
  if (o_out && (!lse_out || (g.W > 0 && (!oc || !oc->o_cache || !oc->lse_cache))))
    return hipErrorInvalidValue;
  StepAttendArgs sa;
  sa.a = make_attend_args(g, step, q_window, c, sel, nullptr, o_ws, l_ws,
                          reinterpret_cast<const char*>(workspace) + g.ws_dummy);
  sa.a.sel_phys = tok_out;  // non-null: the page list carries physical pages (never read here)
  sa.a.tok_k = k_new;
  sa.a.tok_v = v_new;
  sa.scores = reinterpret_cast<float*>((char*)workspace + g.ws_scores);
  sa.A = c.last_loaded;
  sa.tok_out = tok_out;
  sa.err = err;
  sa.k_new = k_new;
  sa.v_new = v_new;
  sa.spin_limit = spin_limit;
  sa.tag_bias = tag_bias;
  sa.m = make_merge_args(g, step, 2, o_ws, l_ws, sel.num_selected, nullptr, nullptr, nullptr,
                         nullptr, oc, o_out, lse_out);
  sa.m.seq_lens = c.seq_lens;
  sa.m.pt = c.page_table;
  sa.lse_tag = reinterpret_cast<uint64_t*>((char*)workspace + g.ws_lse_tag);
  sa.head_tag = reinterpret_cast<uint64_t*>((char*)workspace + g.ws_head_tag);
  const uint32_t nw = (uint32_t)(g.n_splits * g.n_rgroups);
  const uint32_t ppb = (uint32_t)((g.max_pages + (int)nw - 1) / (int)nw);
  const uint32_t grid = (uint32_t)step_attend_workgroups(g);
  uint64_t* tagged = reinterpret_cast<uint64_t*>((char*)workspace + g.ws_tagged);
  uint32_t* ctl = reinterpret_cast<uint32_t*>((char*)workspace + g.ws_heads);
  const uint32_t fp = fingerprint_of(g);
  const uint32_t q_bstride = (uint32_t)((g.W + 1) * g.hq * g.D);
  return dispatch(g, [&](const void*, auto shape, auto t, auto d, auto gc) {
    using T = typename decltype(t)::type;
    using S = decltype(shape);
    constexpr int DD = decltype(d)::value;
    const T* q_cur = reinterpret_cast<const T*>(q_window) + (size_t)g.W * g.hq * g.D;
    step_attend_kernel<T, DD, S::PER, S::SITERS, decltype(gc)::value>
        <<<grid, kThreads, 0, s>>>(reinterpret_cast<T*>(c.digest), (uint32_t)g.max_pages, ppb,
                                   nw, grid, q_cur, (uint32_t)g.hk, q_bstride, ctl, tagged, fp,
                                   sa);
    return hipGetLastError();
  });
}

}  // namespace retro
