// One layer's decode step in a single launch: the dependency graph of Fig. 1 (select
// while speculating, then repair; EMA update beside it) mapped onto workgroup roles of
// one grid instead of two streams.  Roles, in dispatch order (a role only ever waits
// on roles dispatched before it, so every wait ends even when not all workgroups are
// resident at once):
//
//   score    Quest criticality of 128 pages of one KV head (Appendix A.1)
//   select   exact top-K of one KV head (Section 2.1); in the PRR schedule also the
//            missed set A \ P (Section 4.3), attended by this workgroup itself when
//            it holds at most eight pages
//   predict  EMA update with this step's scores and the next predicted set (Eqs. 2-3)
//   spec     attention over a chunk of P, one online-softmax state per page; once A is
//            known the states of the chunk's pages that are in A are folded (Eqs. 6-8),
//            so wasted pages are dropped without any recomputation
//   miss     attention over a chunk of the missed list (serial schedule: of A)
//   merge    merge of every chunk state into the output of one query head (Eqs. 6-8)
//
// Hand-offs inside the launch are 64-bit values {epoch, payload} written with
// device-coherent stores and polled with device-coherent loads: a consumer sees either
// the previous step's epoch or the whole new value, so no counter, flag or fence is
// needed.  The caller passes a new epoch for every call on a workspace.  A select or
// predict workgroup holds 16 keys per thread, so a fused step takes at most 8192 pages.
#pragma once
#include "prr_device.h"
#include "prr_launch.h"
#include "prr_select.h"

namespace prr {


namespace {

constexpr int kFT = 512;
constexpr int kFW = kFT / kWave;
static_assert(kFW == kFusedWaves, "waves per workgroup");
constexpr int kFScorePages = kFusedScorePages;  // pages of one score workgroup
constexpr int kFPagesPerWave = kFScorePages / 8;  // scored by each of its 8 waves
constexpr int kFScoreIt = kFPagesPerWave / 4;     // 4 pages per 16-lane row group at a time
constexpr int kFMaxLists = kFusedMaxPages / kFScorePages;  // score workgroups per KV head
constexpr int kFThreadsPerList = 512 / kFMaxLists;
constexpr int kFSpin = 1 << 20;
constexpr uint32_t kSelfMiss = 0x80000000u;  // missed-list count flags: attended by the select workgroup
constexpr uint32_t kDropSpec = 0x40000000u;  //   the speculation is discarded (recompute on a miss)
constexpr uint32_t kCountMask = 0x3fffffffu;
constexpr int kFOPad = kHeadDim + 4;
constexpr int kEqAll = 16383;  // eq_cut meaning "every key equal to T is taken"
constexpr int kCandMax = 4 * kFT;     // candidates ranked by one workgroup (4 per thread)
constexpr int kCandWave = 12 * kWave;  // candidates ranked by one wave (12 per lane)
// A candidate list of one score workgroup: its tagged count, then its tagged keys; the
// count shares lines with the first keys, and the lists of different workgroups lie in
// different memory channels, so polls of many lists do not queue on one channel.
constexpr int kCandStride = kFScorePages + 4;
// Rank, among this step's candidates, whose key bounds the next step's late pages from
// below: 1.25 |A|.  A lower rank leaves pages of A to the missed list (1.125 |A| does on
// 128K contexts); a higher one attends more pages that turn out not to be in A, and once
// the late pages outnumber what the late workgroups hold the surplus goes to the missed
// list as well.
__host__ __device__ constexpr int kLateRank(int a) { return (5 * a) / 4; }

__device__ __forceinline__ void put_tag(uint64_t* p, uint32_t v, uint32_t epoch) {
  __hip_atomic_store(p, ((uint64_t)epoch << 32) | v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t get_tag(const uint64_t* p) {
  return __hip_atomic_load(const_cast<uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ bool tag_is(uint64_t v, uint32_t epoch) { return (uint32_t)(v >> 32) == epoch; }

// Payload of a tagged value already loaded as v, or, if it is not from this epoch yet,
// of *p once it is (bounded wait; a timeout sets a flag and yields garbage).
__device__ __forceinline__ uint32_t tagged(uint64_t v, const uint64_t* p, uint32_t epoch, uint32_t* flags) {
  for (int it = 0; !tag_is(v, epoch) && it < kFSpin; ++it) {
    __builtin_amdgcn_s_sleep(4);
    v = get_tag(p);
  }
  if (!tag_is(v, epoch)) atomicOr(flags, kFlagSpinTimeout);
  return (uint32_t)v;
}
__device__ __forceinline__ uint32_t wait_tag(const uint64_t* p, uint32_t epoch, uint32_t* flags) {
  return tagged(get_tag(p), p, epoch, flags);
}

// Phase timestamp (called by one thread): the device clock when this workgroup reached
// phase `slot`, one plain store to an entry of its own (only when the caller asked for
// timestamps; workgroups never share an entry, so recording adds no contention).
__device__ __forceinline__ void stamp(const FusedLaunch& a, int slot) {
  if (a.stamps) a.stamps[(size_t)slot * kStampMaxWorkgroups + blockIdx.x] = __builtin_amdgcn_s_memrealtime();
}

// A value that many workgroups wait for (the threshold, the missed and late counts) is
// stored in kRep copies 256 bytes apart, and each waiting workgroup polls one of them, so
// that the polls spread over memory channels instead of queueing on one line.  Record of
// KV head h: kRep copies of kRepStride words; word k of copy c.
constexpr int kRep = 8;
constexpr int kRepStride = 32;
__device__ __forceinline__ uint64_t* rep_at(uint64_t* base, int h, int c) {
  return base + ((size_t)h * kRep + (c & (kRep - 1))) * kRepStride;
}
// stores word k of every copy (one thread)
__device__ __forceinline__ void put_rep(uint64_t* base, int h, int k, uint32_t v, uint32_t epoch) {
#pragma unroll
  for (int c = 0; c < kRep; ++c) put_tag(rep_at(base, h, c) + k, v, epoch);
}

// The threshold record of KV head h (words 0: T, 1: mode | tie cut << 2) and the missed
// count, published in every copy (one thread).
__device__ __forceinline__ void publish_thr(const FusedLaunch& a, int h, uint32_t T, uint32_t me, uint32_t epoch) {
  put_rep(a.t_thr, h, 0, T, epoch);
  put_rep(a.t_thr, h, 1, me, epoch);
  stamp(a, kStampThreshold);
}
__device__ __forceinline__ void publish_mcnt(const FusedLaunch& a, int h, uint32_t v, uint32_t epoch) {
  put_rep(a.t_mcnt, h, 0, v, epoch);
  stamp(a, kStampMissed);
}

// ------------------------------------------------------------------------ LDS

struct FScoreLds {
  float qpart[16][kHeadDim];
  float qbar[kHeadDim];
  float sc[kFScorePages];
  uint32_t fbits[kFScorePages / 32];
};

struct FSelLds {
  union {
    Sel2Lds sel;       // block-wide select
    WSelLds ws[3];     // one-wave selects: A, and the next step's bounds of A and of late pages
    BSelLds bsel;      // threshold of A by the whole workgroup (in place of ws[0])
  };
  uint32_t bitP[PRR_MAX_PAGES_DEV / 32];
  uint32_t forceb[PRR_MAX_PAGES_DEV / 32];
  int32_t mlist[PRR_MAX_CAP_DEV];
  int cnt[2][16];
  int off[3 * kFMaxLists];  // exclusive offsets, counts and forced counts of the score workgroups
  int tot[2];
  float qb[kHeadDim];
  uint32_t ck[kCandMax];
  uint32_t cpg[kCandMax];
  int eq_cut;
  int npv;
};

static_assert(sizeof(BSelLds) <= sizeof(WSelLds), "bsel lies inside ws[0]");

struct FAttnLds {
  float wo[kFW][16][kFOPad];
  float wm[kFW][16];
  float wl[kFW][16];
  int kpg[kFW];     // page of each wave (keep decided after the state is in LDS)
  uint32_t kmask;   // waves whose page is kept
  uint32_t ml[32];  // (m, l) of each row of the combined state
};

struct FMergeLds {
  float red[2][kFW];  // running max and sum of each wave
  float acc[kFW][kHeadDim];
};

struct FLds {
  union {
    FScoreLds score;
    FSelLds sel;
    FAttnLds attn;
    FMergeLds merge;
  };
  // Values polled by one wave and read by the whole workgroup: hundreds of waves
  // polling the same word would queue at its memory channel and slow every hand-off.
  uint32_t bc[2 + 2 * kFW];
  // the G query rows of the KV head (attending roles; never reused within a role)
  u32x4_t qs[16 * kHeadDim / 8];
};
static_assert(sizeof(FLds) <= 80 * 1024, "two workgroups per CU");

// ------------------------------------------------------------------------ score
//
// Besides the scores, a score workgroup filters its pages for the select workgroup: a
// page is a candidate of A when its key reaches the lower bound win[h][0] kept from the
// previous step (or it is forced).  When at least k candidates exist the top-k of all
// pages are among them, so the select workgroup only ranks the candidates; otherwise it
// falls back to all scores.  In the PRR and prefill schedules the workgroup also applies
// the EMA update of Eq. (3) to its pages and filters the next prediction's keys
// (Eq. (2)) the same way, for the predict workgroup.


// EMA of |q-bar|_1 at the rate of the score EMA (the scale of the prediction keys);
// prev = 0: none yet
__device__ __forceinline__ float qn_ema(const FusedLaunch& a, float qn, float prev) {
  return prev > 0.0f ? a.alpha * qn + (1.0f - a.alpha) * prev : qn;
}

template <bool BF16, int PS>
__device__ __forceinline__ void role_score(const FusedLaunch& a, uint32_t ep, int h, int blk, FScoreLds& S) {
  const int t = threadIdx.x, lane = lane_id(), w = t / kWave;
  const int G = a.group;
  const int n = a.num_pages;
  const int pbase = blk * kFScorePages;
  const bool ema = a.schedule != 0;
  const uint16_t* q = static_cast<const uint16_t*>(a.q);
  // wave 0 owns the filtering: EMA state of pages pbase + lane (+ 64 ...)
  constexpr int kHalves = (kFScorePages + kWave - 1) / kWave;
  float lv[kHalves], tv[kHalves];
  uint32_t bw[kHalves];
#pragma unroll
  for (int i = 0; i < kHalves; ++i) {
    lv[i] = tv[i] = 0.f;
    bw[i] = 0u;
  }
  const int nwmax = (a.max_pages + 31) / 32;
  // the query first, then this thread's metadata, so that q-bar is formed while the
  // metadata is still in flight (loads complete in issue order)
  const int g16 = t >> 4, c8 = (t & 15) * 8;
  uint4 qv = make_uint4(0, 0, 0, 0);
  if (g16 < G) qv = *reinterpret_cast<const uint4*>(q + (size_t)(h * G + g16) * kHeadDim + c8);
  const int cg = lane & 15, pi = lane >> 4;
  const int base = pbase + w * kFPagesPerWave + pi;
  uint4 mn[kFScoreIt], mx[kFScoreIt];
  float4 m0[kFScoreIt], m1[kFScoreIt];
  if (!a.meta_mean) {
#pragma unroll
    for (int it = 0; it < kFScoreIt; ++it) {
      const int p = min(base + 4 * it, n - 1);
      const uint16_t* row = static_cast<const uint16_t*>(a.meta) + ((size_t)h * a.max_pages + p) * 2 * kHeadDim + cg * 8;
      mn[it] = *reinterpret_cast<const uint4*>(row);
      mx[it] = *reinterpret_cast<const uint4*>(row + kHeadDim);
    }
  } else {
#pragma unroll
    for (int it = 0; it < kFScoreIt; ++it) {
      const int p = min(base + 4 * it, n - 1);
      const float4* row = reinterpret_cast<const float4*>(static_cast<const float*>(a.meta) +
                                                          ((size_t)h * a.max_pages + p) * kHeadDim + cg * 8);
      m0[it] = row[0];
      m1[it] = row[1];
    }
  }
  // wave 0 filters: EMA state of pages pbase + lane (+ 64 ...), and the
  // candidate bounds kept from the previous step as ratios: of A and of late pages to
  // |q-bar|_1 (scores scale with q-bar), of the next prediction to the EMA of |q-bar|_1
  // (the EMA keys scale with it); loaded together with the metadata
  float r_a = 0.f, r_p = 0.f, r_l = 0.f, qe0 = 0.f;
  uint32_t pw[kHalves];
  int ph[kHalves];  // physical pages (late pages are listed with them)
#pragma unroll
  for (int i = 0; i < kHalves; ++i) {
    pw[i] = 0u;
    ph[i] = 0;
  }
  if (w == 0) {
    r_a = __uint_as_float(a.win[4 * h]);
    r_p = __uint_as_float(a.win[4 * h + 1]);
    r_l = __uint_as_float(a.win[4 * h + 2]);
    qe0 = __uint_as_float(a.win[4 * h + 3]);
    if (a.late) {
#pragma unroll
      for (int half = 0; half < kHalves; ++half) {
        pw[half] = a.pbits_cur[(size_t)h * nwmax + (min(pbase + 64 * half + (lane & 32), n - 1) >> 5)];
        const int p = min(pbase + 64 * half + lane, n - 1);
        ph[half] = a.page_table ? a.page_table[p] : p;
      }
    }
    if (ema) {
#pragma unroll
      for (int half = 0; half < kHalves; ++half) {
        const int p = min(pbase + 64 * half + lane, n - 1);
        lv[half] = a.level[(size_t)h * a.max_pages + p];
        tv[half] = a.trend[(size_t)h * a.max_pages + p];
        bw[half] = a.init_bits[(size_t)h * nwmax + (p >> 5)];
      }
    }
  }
  {
    const int g = g16;
    if (g < G) {
#pragma unroll
      for (int e = 0; e < 8; ++e) S.qpart[g][c8 + e] = u4_elem<BF16>(qv, e);
    }
    if (t < kFScorePages / 32) S.fbits[t] = 0u;
    __syncthreads();
    if (t < kHeadDim) {
      float s = 0.0f;
      for (int gg = 0; gg < G; ++gg) s += S.qpart[gg][t];
      S.qbar[t] = s / (float)G;
    }
    if (t == 0 && a.n_forced > 0) {
      // forced pages of this workgroup's range (the list lives in the kernel arguments:
      // constant indices only)
#pragma unroll
      for (int i = 0; i < PRR_MAX_FORCED; ++i) {
        if (i >= a.n_forced) break;
        const int p = a.forced[i] - pbase;
        if (p >= 0 && p < kFScorePages) S.fbits[p >> 5] |= 1u << (p & 31);
      }
    }
    __syncthreads();
  }
  float qb[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) qb[e] = S.qbar[cg * 8 + e];
  float* scores = a.scores + (size_t)h * a.max_pages;
  uint64_t* ts = a.t_score + (size_t)h * a.max_pages;
  float s[kFScoreIt];
  if (!a.meta_mean) {
#pragma unroll
    for (int it = 0; it < kFScoreIt; ++it) {
      float v = 0.0f;
#pragma unroll
      for (int e = 0; e < 8; ++e) v += fmaxf(qb[e] * u4_elem<BF16>(mn[it], e), qb[e] * u4_elem<BF16>(mx[it], e));
      s[it] = v;
    }
  } else {
#pragma unroll
    for (int it = 0; it < kFScoreIt; ++it) {
      float v = qb[0] * m0[it].x;
      v += qb[1] * m0[it].y;
      v += qb[2] * m0[it].z;
      v += qb[3] * m0[it].w;
      v += qb[4] * m1[it].x;
      v += qb[5] * m1[it].y;
      v += qb[6] * m1[it].z;
      v += qb[7] * m1[it].w;
      s[it] = v;
    }
  }
#pragma unroll
  for (int it = 0; it < kFScoreIt; ++it) {
    const float v = sum16(s[it]);
    const int p = base + 4 * it;
    if (cg == 0) S.sc[p - pbase] = v;
  }
  __syncthreads();
  if (t == 0) stamp(a, kStampScores);
  if (w != 0) return;
  const float qn = wave_sum(fabsf(S.qbar[lane]) + fabsf(S.qbar[lane + 64]));
  const float qe = qn_ema(a, qn, qe0);
  const uint32_t lo_a = score_key(r_a * qn), lo_p = score_key(r_p * qe);
  const uint32_t lo_l = max(score_key(r_l * qn), lo_a);  // late pages are candidates of A

  const size_t rec_a = (size_t)h * a.n_score + blk;
  const size_t rec_p = ((size_t)a.num_kv_heads + h) * a.n_score + blk;
  uint64_t* ck_a = a.t_candk + rec_a * kCandStride + 1;
  uint64_t* cp_a = a.t_candp + rec_a * kFScorePages;
  uint64_t* ck_p = a.t_candk + rec_p * kCandStride + 1;
  uint64_t* cp_p = a.t_candp + rec_p * kFScorePages;
  int na = 0, nfa = 0, np = 0, nfp = 0, nl = 0;
  uint64_t lmask[kHalves];  // late pages of each half
  // Late pages (not forced, not in the bitmap of P^t, key at least lo_l) are listed first:
  // late speculation is the longer chain after the scores.  Then the candidates of A (the
  // select workgroup waits for them), each flagged when it is also a late page, then the
  // EMA update and the candidates of the next prediction.
  const size_t rec_l = (2 * (size_t)a.num_kv_heads + h) * a.n_score + blk;
  uint64_t* ck_l = a.t_candk + rec_l * kCandStride + 1;
  uint64_t* cp_l = a.t_candp + rec_l * kFScorePages;
  bool lt[kHalves];
#pragma unroll
  for (int half = 0; half < kHalves; ++half) {
    lt[half] = false;
    lmask[half] = 0ull;
  }
#pragma unroll
  for (int half = 0; half < kHalves && a.late; ++half) {
    const int lp = 64 * half + lane;
    const int p = pbase + lp;
    const bool inr = p < n && lp < kFScorePages;
    const bool f = inr && ((S.fbits[lp >> 5] >> (lp & 31)) & 1u);
    const uint32_t ka = score_key(S.sc[min(lp, kFScorePages - 1)]);
    const bool late = a.late && inr && !f && ka >= lo_l && !((pw[half] >> (p & 31)) & 1u);
    const uint64_t ml = __ballot(late);
    lt[half] = late;
    lmask[half] = ml;
    if (late) {
      // a late page is listed with its physical page in place of its key (the late
      // workgroups only attend it; the select ranks the candidates of A)
      const int pos = nl + lanes_below(ml);
      put_tag(&ck_l[pos], (uint32_t)ph[half], ep);
      put_tag(&cp_l[pos], (uint32_t)p, ep);
    }
    nl += __popcll(ml);
  }
  if (a.late && lane == 0) put_tag(ck_l - 1, (uint32_t)nl, ep);
#pragma unroll
  for (int half = 0; half < kHalves; ++half) {
    const int lp = 64 * half + lane;
    const int p = pbase + lp;
    const bool inr = p < n && lp < kFScorePages;
    const bool f = inr && ((S.fbits[lp >> 5] >> (lp & 31)) & 1u);
    const float sv = S.sc[min(lp, kFScorePages - 1)];
    if (inr) {
      // the scores, 64 pages per store instruction (whole lines)
      scores[p] = sv;
      put_tag(&ts[p], __float_as_uint(sv), ep);
    }
    const uint32_t ka = score_key(sv);
    const bool ca = inr && (f || ka >= lo_a);
    const bool late = lt[half];
    const uint64_t ma = __ballot(ca), mfa = __ballot(ca && f);
    if (ca) {
      const int pos = na + lanes_below(ma);
      put_tag(&ck_a[pos], ka, ep);
      put_tag(&cp_a[pos], (uint32_t)p | (f ? 0x80000000u : 0u) | (late ? 0x40000000u : 0u), ep);
    }
    na += __popcll(ma);
    nfa += __popcll(mfa);
  }
  if (lane == 0) put_tag(ck_a - 1, (uint32_t)na | ((uint32_t)nfa << 16), ep);
  if (a.stamps) {
    stores_complete();
    if (lane == 0) stamp(a, kStampCandidates);
  }
  // The K and V of the first late pages, one word per 64-byte line, read now: the late
  // workgroups load them about two microseconds later and then find them in the
  // memory-side cache.  The words only feed a check at the end of this role.
  constexpr int kPfLoads = PS * kHeadDim * 2 / (64 * kWave);  // instructions per K (or V) of a page
  constexpr int kPfPages = 8;
  uint32_t pf[kPfPages][2 * kPfLoads];
#pragma unroll
  for (int k = 0; k < kPfPages; ++k) {
#pragma unroll
    for (int j = 0; j < 2 * kPfLoads; ++j) pf[k][j] = 0u;
  }
  if (a.readahead) {
    const char* kh = static_cast<const char*>(a.k_cache) + (size_t)h * a.max_pages * PS * kHeadDim * 2;
    const char* vh = static_cast<const char*>(a.v_cache) + (size_t)h * a.max_pages * PS * kHeadDim * 2;
    uint64_t m0 = lmask[0], m1 = kHalves > 1 ? lmask[kHalves - 1] : 0ull;
#pragma unroll
    for (int k = 0; k < kPfPages; ++k) {
      int q = -1;
      if (m0) {
        const int l = __builtin_ctzll(m0);
        m0 &= m0 - 1;
        q = __builtin_amdgcn_readlane(ph[0], l);
      } else if (m1) {
        const int l = __builtin_ctzll(m1);
        m1 &= m1 - 1;
        q = __builtin_amdgcn_readlane(ph[kHalves - 1], l);
      }
      if (q >= 0 && q < a.max_pages) {
        const size_t page = (size_t)q * PS * kHeadDim * 2;
#pragma unroll
        for (int j = 0; j < kPfLoads; ++j) {
          const size_t o = page + ((size_t)j * kWave + lane) * 64;
          pf[k][j] = *reinterpret_cast<const uint32_t*>(kh + o);
          pf[k][kPfLoads + j] = *reinterpret_cast<const uint32_t*>(vh + o);
        }
      }
    }
  }
  if (!ema) return;
  // ... then the EMA update of Eq. (3) and the candidates of the next prediction
#pragma unroll
  for (int half = 0; half < kHalves; ++half) {
    const int lp = 64 * half + lane;
    const int p = pbase + lp;
    const bool inr = p < n && lp < kFScorePages;
    const float sv = S.sc[min(lp, kFScorePages - 1)];
    const bool f = inr && ((S.fbits[lp >> 5] >> (lp & 31)) & 1u);
    bool has = inr && ((bw[half] >> (p & 31)) & 1u);
    float l = lv[half], v = tv[half];
    if (inr) {
      if (has) {
        v = a.beta * (sv - l) + (1.0f - a.beta) * v;  // Eq. (3): the trend reads the previous level
        l = a.alpha * sv + (1.0f - a.alpha) * l;
      } else {
        l = sv;
        v = 0.0f;
        has = true;
      }
      a.level[(size_t)h * a.max_pages + p] = l;
      a.trend[(size_t)h * a.max_pages + p] = v;
    }
    const uint64_t hm = __ballot(has), vm = __ballot(inr);
    if (lane == 0 || lane == 32) {
      const uint32_t hbits = (uint32_t)(lane == 0 ? hm : (hm >> 32));
      const uint32_t vbits = (uint32_t)(lane == 0 ? vm : (vm >> 32));
      if (vbits) a.init_bits[(size_t)h * nwmax + (p >> 5)] = (bw[half] & ~vbits) | hbits;
    }
    const uint32_t kp = score_key(l + a.gamma * v);  // Eq. (2)
    if (inr) put_tag(&a.t_pkey[(size_t)h * a.max_pages + p], kp, ep);
    const bool cpred = inr && (f || kp >= lo_p);
    const uint64_t mp = __ballot(cpred), mfp = __ballot(cpred && f);
    if (cpred) {
      const int pos = np + lanes_below(mp);
      put_tag(&ck_p[pos], kp, ep);
      put_tag(&cp_p[pos], (uint32_t)p | (f ? 0x80000000u : 0u), ep);
    }
    np += __popcll(mp);
    nfp += __popcll(mfp);
  }
  if (lane == 0) put_tag(ck_p - 1, (uint32_t)np | ((uint32_t)nfp << 16), ep);
  uint32_t px = 0u;
#pragma unroll
  for (int k = 0; k < kPfPages; ++k) {
#pragma unroll
    for (int j = 0; j < 2 * kPfLoads; ++j) px ^= pf[k][j];
  }
  if (px == ep * 2654435761u + 0x9e3779b9u) atomicOr(a.flags, 0u);  // (no effect when it holds)
}

// ------------------------------------------------------------------------ shared select pieces

__device__ __forceinline__ bool bit_of(const uint32_t* bits, int p) { return (bits[p >> 5] >> (p & 31)) & 1u; }

// ------------------------------------------------------------------------ attention

// One wave's pages (wave-uniform logical ids, -1 = none): an online-softmax state per page.
// Lane 16j+n holds the state of query head n; acc[k][cb][i] is the unnormalised output
// channel 32j + 8i + cb of head n, m[k] the page's maximum scaled logit, l[k] its sum.
template <int NPW>
struct WaveStates {
  f32x4_t acc[NPW][8];
  float m[NPW];
  float l[NPW];
};

template <bool BF16>
__device__ __forceinline__ f32x4_t mfma_qk(const u32x4_t& x, const u32x4_t& y, f32x4_t c) {
  if constexpr (BF16) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, x), __builtin_bit_cast(bf16x8_t, y), c,
                                                   0, 0, 0);
  } else {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8_t, x), __builtin_bit_cast(f16x8_t, y), c, 0,
                                                  0, 0);
  }
}

// q.k^T of a 16-token tile as four 16x16x32 MFMAs with the contraction index permuted so
// that lane 16j+r reads 64 contiguous bytes of its key row (channels 32j..32j+31); the
// result gives lane 16j+n the logits of tokens 4j..4j+3 for head n.  p.V is computed
// transposed, O^T += V^T P^T, by pv_tile (prr_device.h): lane 16j+m supplies channel
// 8m+cb of V rows 4j..4j+3 and the weights of head m for those tokens.
// Query fragments of KV head h for the MFMA layout below (lane 16j+n: head n, channels
// 32j..32j+31), loaded before a workgroup waits for its page list.
// The MFMA operand fragments of q (G rows of the KV head): the rows are read from memory
// once per workgroup into LDS and the waves take their fragments from there.  Eight
// waves each reading the whole of q put eight times the traffic through the CU's memory
// pipeline at the launch's start, where the attending workgroups share CUs with score
// workgroups that are still reading metadata.  Called by every thread (one barrier).
// this lane's MFMA operand of q (query head n of the group, channels 32j + 8s ..) from the
// rows staged in LDS
__device__ __forceinline__ void fetch_q(const FusedLaunch& a, u32x4_t (&qf)[4], const u32x4_t* qs) {
  const int lane = lane_id(), j = lane >> 4, n = lane & 15;
  constexpr int kRow = kHeadDim / 8;  // 16-byte words per row
  if (n < a.group) {
#pragma unroll
    for (int s = 0; s < 4; ++s) qf[s] = qs[n * kRow + 4 * j + s];
  } else {
#pragma unroll
    for (int s = 0; s < 4; ++s) qf[s] = u32x4_t{0, 0, 0, 0};
  }
}

__device__ __forceinline__ void load_q(const FusedLaunch& a, int h, u32x4_t (&qf)[4], u32x4_t* qs) {
  const int t = threadIdx.x;
  const int G = a.group;
  constexpr int kRow = kHeadDim / 8;
  const u32x4_t* qh = reinterpret_cast<const u32x4_t*>(static_cast<const uint16_t*>(a.q) + (size_t)h * G * kHeadDim);
  if (t < G * kRow) qs[t] = qh[t];
  __syncthreads();
  fetch_q(a, qf, qs);
}

template <bool BF16, int PS, int NPW>
__device__ __forceinline__ void wave_attend(const FusedLaunch& a, int h, const u32x4_t (&qf)[4], const int (&pg)[NPW],
                                            WaveStates<NPW>& st, const int* phys_in = nullptr) {
  constexpr int TPP = PS / 16;
  constexpr int NTW = NPW * TPP;
  const float kNegInf = -__builtin_inff();
  const float scale = 0.08838834764831845f;  // 1/sqrt(128)
  const int lane = lane_id(), j = lane >> 4, n = lane & 15;
  const uint16_t* kh = static_cast<const uint16_t*>(a.k_cache) + (size_t)h * a.max_pages * PS * kHeadDim;
  const uint16_t* vh = static_cast<const uint16_t*>(a.v_cache) + (size_t)h * a.max_pages * PS * kHeadDim;
  int phys[NPW];
#pragma unroll
  for (int k = 0; k < NPW; ++k)
    phys[k] = phys_in ? phys_in[k] : ((pg[k] >= 0 && a.page_table) ? a.page_table[pg[k]] : pg[k]);
  bool ok[NPW];
  size_t off[NPW];
#pragma unroll
  for (int k = 0; k < NPW; ++k) {
    const int ph = __builtin_amdgcn_readfirstlane(phys[k]);
    ok[k] = pg[k] >= 0 && ph >= 0 && ph < a.max_pages;
    if (pg[k] >= 0 && !ok[k] && lane == 0) atomicOr(a.flags, kFlagBadListEntry);
    off[k] = ok[k] ? (size_t)ph * PS * kHeadDim : 0;
  }
  u32x4_t kf[NTW][4], vf[NTW][4];
#pragma unroll
  for (int f = 0; f < NTW; ++f) {
    const int k = f / TPP, tt = f % TPP;
    if (ok[k]) {
      const uint16_t* kt = kh + off[k] + (size_t)tt * 16 * kHeadDim;
      const uint16_t* vt = vh + off[k] + (size_t)tt * 16 * kHeadDim;
      const u32x4_t* ks = reinterpret_cast<const u32x4_t*>(kt + (size_t)n * kHeadDim + 32 * j);
#pragma unroll
      for (int s = 0; s < 4; ++s) kf[f][s] = ks[s];
#pragma unroll
      for (int tg = 0; tg < 4; ++tg)
        vf[f][tg] = *reinterpret_cast<const u32x4_t*>(vt + (size_t)(4 * j + tg) * kHeadDim + 8 * n);
    }
  }
#pragma unroll
  for (int k = 0; k < NPW; ++k) {
#pragma unroll
    for (int cb = 0; cb < 8; ++cb) st.acc[k][cb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    st.m[k] = kNegInf;
    st.l[k] = 0.0f;
  }
#pragma unroll
  for (int f = 0; f < NTW; ++f) {
    const int k = f / TPP, tt = f % TPP;
    if (!ok[k]) continue;
    f32x4_t sc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < 4; ++s) sc = mfma_qk<BF16>(kf[f][s], qf[s], sc);
    float sv[4];
    float mx = kNegInf;
    const int tok0 = pg[k] * PS + tt * 16 + 4 * j;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      sv[i] = (tok0 + i) < a.num_tokens ? sc[i] * scale : kNegInf;
      mx = fmaxf(mx, sv[i]);
    }
    mx = max_rows(mx);
    const float mnew = fmaxf(st.m[k], mx);
    float alpha = 1.0f;
    float p[4] = {0.f, 0.f, 0.f, 0.f};
    if (mnew != kNegInf) {
      alpha = exp2f((st.m[k] - mnew) * kLog2e);
#pragma unroll
      for (int i = 0; i < 4; ++i) p[i] = exp2f((sv[i] - mnew) * kLog2e);
    }
    const float ls = sum_rows((p[0] + p[1]) + (p[2] + p[3]));
    st.l[k] = st.l[k] * alpha + ls;
    st.m[k] = mnew;
    if (pg[k] * PS + PS > a.num_tokens) {
      // a partial last page: the values of tokens at or past num_tokens are zeroed, not
      // only weighted by 0 (0 x NaN or Inf from an unwritten cache tail would poison o)
#pragma unroll
      for (int tg = 0; tg < 4; ++tg)
        if (tok0 + tg >= a.num_tokens) vf[f][tg] = u32x4_t{0, 0, 0, 0};
    }
    if (tt > 0) {
#pragma unroll
      for (int cb = 0; cb < 8; ++cb) {
#pragma unroll
        for (int i = 0; i < 4; ++i) st.acc[k][cb][i] *= alpha;
      }
    }
    pv_tile<BF16>(st.acc[k], vf[f], p);
  }
}

// Where a workgroup publishes its partial state (slot `slot` of KV head h), computed
// before a long wait and kept in scalar registers: the kernel arguments it derives
// from would otherwise be loaded again after the wait, on the critical path.
struct PubDst {
  float* po;      // [G][128] outputs of the slot
  uint64_t* pml;  // [G][2] tagged (m, l) of the slot
  int G;
};
__device__ __forceinline__ PubDst pub_dst(const FusedLaunch& a, int h, int slot) {
  const size_t row0 = ((size_t)h * a.nparts + slot) * a.group;
  const uint64_t po = (uint64_t)(a.part_o + row0 * kHeadDim), pml = (uint64_t)(a.t_part + row0 * 2);
  uint32_t w[5] = {(uint32_t)po, (uint32_t)(po >> 32), (uint32_t)pml, (uint32_t)(pml >> 32), (uint32_t)a.group};
#pragma unroll
  for (int i = 0; i < 5; ++i) {
    w[i] = (uint32_t)__builtin_amdgcn_readfirstlane((int)w[i]);
    asm volatile("" : "+s"(w[i]));
  }
  PubDst d;
  d.po = reinterpret_cast<float*>((uint64_t)w[0] | ((uint64_t)w[1] << 32));
  d.pml = reinterpret_cast<uint64_t*>((uint64_t)w[2] | ((uint64_t)w[3] << 32));
  d.G = (int)w[4];
  return d;
}

// Fold the kept page states of this wave (keep: wave-uniform bit mask) and write the
// result to the wave's LDS slot.
template <int NPW>
__device__ __forceinline__ void fold_write(WaveStates<NPW>& st, uint32_t keep, FAttnLds& L) {
  const float kNegInf = -__builtin_inff();
  const int lane = lane_id(), w = threadIdx.x / kWave;
  const int j = lane >> 4, n = lane & 15;
  float mf = kNegInf;
#pragma unroll
  for (int k = 0; k < NPW; ++k)
    if (((keep >> k) & 1u) && st.l[k] > 0.0f) mf = fmaxf(mf, st.m[k]);
  float lf = 0.0f;
  f32x4_t acc[8];
#pragma unroll
  for (int cb = 0; cb < 8; ++cb) acc[cb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int k = 0; k < NPW; ++k) {
    if (((keep >> k) & 1u) && st.l[k] > 0.0f) {
      const float f = exp2f((st.m[k] - mf) * kLog2e);
      lf += st.l[k] * f;
#pragma unroll
      for (int cb = 0; cb < 8; ++cb) {
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[cb][i] += st.acc[k][cb][i] * f;
      }
    }
  }
  if (j == 0) {
    L.wm[w][n] = mf;
    L.wl[w][n] = lf;
  }
  float* row = &L.wo[w][n][32 * j];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    *reinterpret_cast<float4*>(row + 8 * i) = make_float4(acc[0][i], acc[1][i], acc[2][i], acc[3][i]);
    *reinterpret_cast<float4*>(row + 8 * i + 4) = make_float4(acc[4][i], acc[5][i], acc[6][i], acc[7][i]);
  }
}

// The states of the waves in `wmask` (uniform) combined per row and published (the
// states are in LDS, behind a barrier).
__device__ __forceinline__ void combine_publish(const FusedLaunch& a, int slot, const PubDst& d, uint32_t ep,
                                                uint32_t wmask, FAttnLds& L) {
  const float kNegInf = -__builtin_inff();
  const int t = threadIdx.x, lane = lane_id();
  const int hh = t >> 5, ci = t & 31;  // row; columns 2ci, 2ci + 1, 64 + 2ci, 65 + 2ci
  const int G = d.G;
  static_assert(kFW == 8, "the weights of a row are spread over 8 lanes");
  // The weight of wave ww's state for this row is computed once, by lane ww of the row's
  // 32-lane group (lanes repeat it every 8), and read from there: the fold's arithmetic
  // runs on every wave of the CU at once, so its instruction count is its latency.
  const int ww8 = lane & 7;
  const float mv = hh < G ? L.wm[ww8][hh] : kNegInf;
  const float lv = (hh < G && ((wmask >> ww8) & 1u)) ? L.wl[ww8][hh] : 0.0f;
  float ms = lv > 0.0f ? mv : kNegInf;
  ms = fmaxf(ms, dpp_f32<kDppXor1>(ms));
  ms = fmaxf(ms, dpp_f32<kDppXor2>(ms));
  ms = fmaxf(ms, dpp_f32<kDppHalfMirror>(ms));
  const float fwl = lv > 0.0f ? exp2f((mv - ms) * kLog2e) : 0.0f;
  float lsum = lv * fwl;
  lsum += dpp_f32<kDppXor1>(lsum);
  lsum += dpp_f32<kDppXor2>(lsum);
  lsum += dpp_f32<kDppHalfMirror>(lsum);
  if (hh < G) {
    const float inv = lsum > 0.0f ? 1.0f / lsum : 0.0f;
    const int hi = lane & 32;
    float o[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ww = 0; ww < kFW; ++ww) {
      const float f0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(fwl), ww));
      const float f1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(fwl), 32 + ww));
      const float f = hi ? f1 : f0;
      const float2 xa = *reinterpret_cast<const float2*>(&L.wo[ww][hh][2 * ci]);
      const float2 xb = *reinterpret_cast<const float2*>(&L.wo[ww][hh][64 + 2 * ci]);
      o[0] += xa.x * f;
      o[1] += xa.y * f;
      o[2] += xb.x * f;
      o[3] += xb.y * f;
    }
    // each store instruction of a wave covers whole lines (partial lines written
    // through to memory cost a read-modify-write each)
    uint64_t* dst = reinterpret_cast<uint64_t*>(d.po + (size_t)hh * kHeadDim);
    const uint64_t va = (uint64_t)__float_as_uint(o[0] * inv) | ((uint64_t)__float_as_uint(o[1] * inv) << 32);
    const uint64_t vb = (uint64_t)__float_as_uint(o[2] * inv) | ((uint64_t)__float_as_uint(o[3] * inv) << 32);
    __hip_atomic_store(dst + ci, va, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(dst + 32 + ci, vb, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if ((t & 31) == 0) {
      L.ml[2 * hh] = __float_as_uint(lsum > 0.0f ? ms : kNegInf);
      L.ml[2 * hh + 1] = __float_as_uint(lsum);
    }
  }
  // The tagged (m, l) of a state are stored only after every output value of it has
  // completed (device-coherent stores are acknowledged once visible to the whole
  // device), so a reader that sees them current reads a complete, untagged output;
  // all rows' (m, l) go out in one store instruction.
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (t < 2 * G) put_tag(d.pml + t, L.ml[t], ep);
  if (t == 0) stamp(a, slot);
}

// Fold the kept page states of every wave (keep: wave-uniform bit mask) and publish the
// workgroup's state.
template <int NPW>
__device__ __forceinline__ void fold_publish(const FusedLaunch& a, int slot, const PubDst& d, uint32_t ep,
                                             WaveStates<NPW>& st, uint32_t keep, FAttnLds& L) {
  fold_write<NPW>(st, keep, L);
  __syncthreads();
  combine_publish(a, slot, d, ep, 0xffu, L);
}

__device__ __forceinline__ bool page_forced(const FusedLaunch& a, int p) {
  bool f = false;
#pragma unroll
  for (int i = 0; i < PRR_MAX_FORCED; ++i) {
    if (i >= a.n_forced) break;
    f |= a.forced[i] == p;
  }
  return f;
}

// ------------------------------------------------------------------------ select

// Candidates of list `which` (0: A, 1: the next P) of KV head h.  Thread t serves score
// workgroup t / 8: it loads that workgroup's count together with the workgroup's
// entries t % 8 and t % 8 + 8 (most workgroups have fewer than 16 candidates, so one
// round trip usually brings everything), then the list is laid out in LDS in page
// order (exclusive offsets of the workgroups by a wave prefix sum).
struct FCand {
  int total, nforced;
};

// POLL_ALL: every thread polls (the count and the first entries of one score workgroup
// per kFThreadsPerList threads: one round trip after the last list, used by the select
// workgroup); otherwise one wave polls the counts and the entries are loaded afterwards,
// a light poll for the many late-speculation workgroups and for the predict workgroup
// (polling every list's entries from all of them measured slower).
template <bool POLL_ALL>
__device__ __forceinline__ FCand cand_load(const FusedLaunch& a, uint32_t ep, int h, int which, int* off, int* tot, uint32_t* lk,
                                           uint32_t* lp) {
  constexpr int TPL = kFThreadsPerList;  // threads per list
  constexpr int L2 = kFMaxLists / kWave; // lists per lane in the one-wave paths
  static_assert(TPL * kFMaxLists == 512 && L2 * kWave == kFMaxLists, "list layout");
  int* cnt = off + kFMaxLists;
  int* fcnt = off + 2 * kFMaxLists;
  const int t = threadIdx.x, lane = lane_id(), w = t / kWave;
  const int nS = a.n_score;
  const int wg = t / TPL, sub = t % TPL;
  const bool mine = wg < nS;
  const size_t rec0 = ((size_t)which * a.num_kv_heads + h) * nS;
  const size_t rec = rec0 + min(wg, nS - 1);
  const uint64_t* ck = a.t_candk + rec * kCandStride + 1;
  const uint64_t* cp = a.t_candp + rec * kFScorePages;
  // the count and the first two entries per thread are polled together until all
  // needed are there (16 per list, more than most lists hold; the rest of a longer list
  // is loaded after the poll)
  constexpr int kPollE = 16 / TPL;
  uint64_t vc = 0, ke[kPollE], pe[kPollE];
#pragma unroll
  for (int u = 0; u < kPollE; ++u) ke[u] = pe[u] = 0ull;
  uint32_t c = 0u;
  if (!POLL_ALL && w == 0) {
    // lane l polls the counts of lists l, l + 64, ..
    uint64_t v[L2];
    for (int it = 0; it < kFSpin; ++it) {
      bool missing = false;
#pragma unroll
      for (int k = 0; k < L2; ++k) {
        const int li = lane + kWave * k;
        v[k] = get_tag(&a.t_candk[(rec0 + min(li, nS - 1)) * kCandStride]);
        missing = missing || (li < nS && !tag_is(v[k], ep));
      }
      if (__ballot(missing) == 0ull) break;
      __builtin_amdgcn_s_sleep(2);
      if (it == kFSpin - 1 && lane == 0) atomicOr(a.flags, kFlagSpinTimeout);
    }
#pragma unroll
    for (int k = 0; k < L2; ++k) {
      const int li = lane + kWave * k;
      if (li < nS) {
        cnt[li] = (int)((uint32_t)v[k] & 0xffffu);
        fcnt[li] = (int)((uint32_t)v[k] >> 16);
      }
    }
  }
  for (int it = 0; POLL_ALL && mine && it < kFSpin; ++it) {
    vc = get_tag(ck - 1);
#pragma unroll
    for (int u = 0; u < kPollE; ++u) {
      ke[u] = get_tag(&ck[sub + TPL * u]);
      pe[u] = get_tag(&cp[sub + TPL * u]);
    }
    if (tag_is(vc, ep)) {
      c = (uint32_t)vc;
      const int n0 = (int)(c & 0xffffu);
      bool ok = true;
#pragma unroll
      for (int u = 0; u < kPollE; ++u)
        ok = ok && (sub + TPL * u >= n0 || (tag_is(ke[u], ep) && tag_is(pe[u], ep)));
      if (ok) break;
    }
    __builtin_amdgcn_s_sleep(2);
    if (it == kFSpin - 1) atomicOr(a.flags, kFlagSpinTimeout);
  }
  if (POLL_ALL && mine && sub == 0) {
    cnt[wg] = (int)(c & 0xffffu);
    fcnt[wg] = (int)(c >> 16);
  }
  __syncthreads();
  const int nc = mine ? cnt[wg] : 0;
  if (w == 0) {
    // lane l holds lists L2 l .. L2 l + L2 - 1 (consecutive, so the offsets follow a scan)
    int cw[L2], sum = 0, fs = 0;
#pragma unroll
    for (int k = 0; k < L2; ++k) {
      const int li = L2 * lane + k;
      cw[k] = li < nS ? cnt[li] : 0;
      sum += cw[k];
      fs += li < nS ? fcnt[li] : 0;
    }
    const int incl = wave_inclusive_scan(sum);
    int o = incl - sum;
#pragma unroll
    for (int k = 0; k < L2; ++k) {
      const int li = L2 * lane + k;
      if (li < nS) off[li] = o;
      o += cw[k];
    }
    const int ft = wave_isum(fs);
    if (lane == kWave - 1) {
      tot[0] = incl;
      tot[1] = ft;
    }
  }
  __syncthreads();
  FCand r;
  r.total = tot[0];
  r.nforced = tot[1];
  if (mine && r.total <= kCandMax) {
    const int o = off[wg];
    if (POLL_ALL) {
      // the poll above only ended once every one of these slots below the count was
      // from this epoch
#pragma unroll
      for (int u = 0; u < kPollE; ++u) {
        const int slot = sub + TPL * u;
        if (slot < nc) {
          lk[o + slot] = (uint32_t)ke[u];
          lp[o + slot] = (uint32_t)pe[u];
        }
      }
    }
    // the rest in batches of four per thread, all loads of a batch issued before any wait
    for (int s0 = sub + (POLL_ALL ? TPL * kPollE : 0); s0 < nc; s0 += 4 * TPL) {
      uint64_t kv[4], pv[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int slot = min(s0 + TPL * u, kFScorePages - 1);
        kv[u] = get_tag(&ck[slot]);
        pv[u] = get_tag(&cp[slot]);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int slot = s0 + TPL * u;
        if (slot < nc) {
          lk[o + slot] = tagged(kv[u], &ck[slot], ep, a.flags);
          lp[o + slot] = tagged(pv[u], &cp[slot], ep, a.flags);
        }
      }
    }
  }
  __syncthreads();
  return r;
}

// The candidate list (LDS, page order) into this thread's slots i = (w, j, lane).
template <int J>
__device__ __forceinline__ void cand_slots(int total, const uint32_t* lk, const uint32_t* lp, uint32_t (&key)[J],
                                           int (&page)[J], uint64_t& cand, uint64_t& force, uint64_t* late) {
  cand = 0;
  force = 0;
  uint64_t lb = 0;
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int i = sel2_page<J>(j);
    key[j] = 0u;
    page[j] = 0;
    if (i < total) {
      key[j] = lk[i];
      const uint32_t pv = lp[i];
      page[j] = (int)(pv & 0x3fffffffu);
      if (pv >> 31) force |= 1ull << j;
      else cand |= 1ull << j;
      if ((pv >> 30) & 1u) lb |= 1ull << j;
    }
  }
  if (late) *late = lb;
}

// All pages of KV head h as slots (the fallback): keys polled from `tk`.
template <int J>
__device__ __forceinline__ void full_gather(const FusedLaunch& a, uint32_t ep, const uint64_t* tk, const uint32_t* forceb,
                                            uint32_t (&key)[J], int (&page)[J], uint64_t& cand, uint64_t& force) {
  const int n = a.num_pages;
  uint64_t pending = 0;
#pragma unroll
  for (int j = 0; j < J; ++j) {
    key[j] = 0u;
    page[j] = sel2_page<J>(j);
    if (page[j] < n) pending |= 1ull << j;
  }
  for (int it = 0; pending && it < kFSpin; ++it) {
    uint64_t v[J];
#pragma unroll
    for (int j = 0; j < J; ++j) v[j] = get_tag(&tk[min(page[j], n - 1)]);
#pragma unroll
    for (int j = 0; j < J; ++j) {
      if (((pending >> j) & 1ull) && tag_is(v[j], ep)) {
        key[j] = (uint32_t)v[j];
        pending &= ~(1ull << j);
      }
    }
    if (pending) __builtin_amdgcn_s_sleep(4);
  }
  if (pending) atomicOr(a.flags, kFlagSpinTimeout);
  cand = 0;
  force = 0;
#pragma unroll
  for (int j = 0; j < J; ++j) {
    if (page[j] >= n) continue;
    if (bit_of(forceb, page[j])) force |= 1ull << j;
    else cand |= 1ull << j;
  }
}

// Lower bound of the next step's candidates: the score of rank `k` (2.25 |A| for the
// candidates, 1.25 |A| for late speculation) among this step's candidates, kept as a
// ratio to |q-bar|_1 (unchanged when fewer candidates exist and `keep` is set; -inf,
// i.e. every page, after a fallback that found fewer).
__device__ __forceinline__ float key_value(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

template <int J>
__device__ __forceinline__ void update_window(const FusedLaunch& a, uint32_t* win, float qn, const uint32_t (&key)[J],
                                              uint64_t cand, int k, bool keep, Sel2Lds& S) {
  __syncthreads();  // the LDS may still be read by the previous step of this workgroup
  const SelThreshold th = sel2_threshold<kFT, J>(key, cand, max(k, 1), S);
  if (threadIdx.x == 0) {
    if (th.mode == 2 && qn > 0.0f) *win = __float_as_uint(key_value(th.T) / qn);
    else if (!keep) *win = __float_as_uint(-__builtin_inff());
  }
}

// |q-bar_h|_1 (every thread), with q-bar as the score workgroups compute it: channel t
// of the G query heads loaded by thread t < 128, summed in head order.
template <bool BF16>
__device__ __forceinline__ void qbar_load(const FusedLaunch& a, int h, float (&qv)[16]) {
  const int t = threadIdx.x;
  const int G = a.group;
  const uint16_t* q = static_cast<const uint16_t*>(a.q) + (size_t)h * G * kHeadDim;
#pragma unroll
  for (int g = 0; g < 16; ++g) qv[g] = (t < kHeadDim && g < G) ? h2f<BF16>(q[(size_t)g * kHeadDim + t]) : 0.0f;
}
__device__ __forceinline__ float qbar_finish(const FusedLaunch& a, const float (&qv)[16], float* qb) {
  const int t = threadIdx.x;
  if (t < kHeadDim) {
    float s = 0.0f;
#pragma unroll
    for (int g = 0; g < 16; ++g)
      if (g < a.group) s += qv[g];
    qb[t] = fabsf(s / (float)a.group);
  }
  __syncthreads();
  return wave_sum(qb[lane_id()] + qb[lane_id() + 64]);
}

template <bool BF16, int PS, int J>
__device__ __forceinline__ void select_finish(const FusedLaunch& a, uint32_t ep, int h, const uint32_t (&key)[J],
                                              const int (&page)[J], uint64_t cand, uint64_t force, uint64_t late_bits,
                                              bool keep_window, float qn, FLds& U) {
  FSelLds& L = U.sel;
  const int t = threadIdx.x, lane = lane_id(), w = t / kWave;
  const bool prr = a.schedule == 1;
  uint64_t inP = 0;
  if (prr) {
#pragma unroll
    for (int j = 0; j < J; ++j)
      if ((((cand | force) >> j) & 1ull) && bit_of(L.bitP, page[j])) inP |= 1ull << j;
  }
  const SelThreshold th = sel2_threshold<kFT, J>(key, cand, a.kextra_a, L.sel);
  const bool early = th.mode != 2 || th.need_eq >= th.eq_total;
  if (prr && early && t == 0) {
    publish_thr(a, h, th.T, (uint32_t)th.mode | ((uint32_t)kEqAll << 2), ep);
  }
  const uint64_t inA = sel2_membership<kFT, J>(key, page, cand, force, th, &L.eq_cut, L.sel);
  if (prr && !early) {
    __syncthreads();
    if (t == 0) {
      publish_thr(a, h, th.T, (uint32_t)th.mode | ((uint32_t)L.eq_cut << 2), ep);
    }
  }

  // pages attended by late speculation: flagged candidates within the late capacity
  // (rank among the flagged pages in page order), never a page of P^t
  uint64_t inLate = 0;
  if (a.late) {
    uint64_t flagged = 0;
#pragma unroll
    for (int j = 0; j < J; ++j)
      if ((((cand | force) >> j) & 1ull) && (late_bits >> j) & 1ull) flagged |= 1ull << j;
    const int lc = wave_isum(__popcll(flagged));
    __syncthreads();
    if (lane == 0) L.cnt[0][w] = lc;
    __syncthreads();
    int run = 0, ltot = 0;
#pragma unroll
    for (int i = 0; i < kFW; ++i) {
      run += i < w ? L.cnt[0][i] : 0;
      ltot += L.cnt[0][i];
    }
    const int capl = a.n_late * a.chunk;
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const bool f = (flagged >> j) & 1ull;
      const uint64_t bm = __ballot(f);
      if (f && run + lanes_below(bm) < capl && !((inP >> j) & 1ull)) inLate |= 1ull << j;
      run += __popcll(bm);
    }
    if (t == 0) put_rep(a.t_lcnt, h, 0, (uint32_t)min(ltot, capl), ep);
  }
  // the list to attend after selection, in page order: A \ P (PRR; also without the
  // late-speculated pages) or A (serial, or a PRR step whose speculation is discarded
  // because a page was missed)
  const int nMiss = prr ? block_sum<kFT>(__popcll(inA & ~inP), L.sel.red[2]) : 0;
  const bool drop = prr && a.mode == PRR_RECOMPUTE_ON_MISS && nMiss > 0;
  const uint64_t inM = (prr && !drop) ? (inA & ~inP & ~inLate) : inA;
  const uint32_t mflags = drop ? kDropSpec : 0u;
  const int nM = min(sel2_list<kFT, J>(inM, page, L.mlist, a.cap, L.sel), a.cap);
  __syncthreads();
  if (nM == 0) {
    if (t == 0) publish_mcnt(a, h, mflags, ep);
  } else if (nM > kFW) {
    uint64_t* ml = a.t_mlist + (size_t)h * a.cap;
    for (int i = t; i < nM; i += kFT) put_tag(&ml[i], (uint32_t)L.mlist[i], ep);
    if (t == 0) publish_mcnt(a, h, (uint32_t)nM | mflags, ep);
  }
  // the selected list (an output) and the counts
  int32_t* sel = a.selected + (size_t)h * a.cap;
  int nA;
  if (prr && !drop) {
    nA = min(sel2_list<kFT, J>(inA, page, sel, a.cap, L.sel), a.cap);
  } else {
    nA = nM;
    for (int i = t; i < nM; i += kFT) sel[i] = L.mlist[i];
  }
  const int nPA = prr ? block_sum<kFT>(__popcll(inP & inA), L.sel.red[2]) : 0;
  if (t == 0) {
    a.selected_count[h] = nA;
    if (a.missed_count) a.missed_count[h] = prr ? nMiss : nM;
    if (a.wasted_count) a.wasted_count[h] = prr ? L.npv - nPA : 0;
    if (a.covered_count) a.covered_count[h] = prr ? max(nMiss - nM, 0) : 0;  // (0 when M = A)
  }
  if (nM > 0 && nM <= kFW) {
    // few enough to attend here: one page per wave, published as the first miss slot
    if (t == 0) publish_mcnt(a, h, (uint32_t)nM | kSelfMiss | mflags, ep);
    int pg[1];
    pg[0] = __builtin_amdgcn_readfirstlane(w < nM ? L.mlist[w] : -1);
    __syncthreads();  // the list is read before the attention reuses the LDS
    u32x4_t qf[4];
    load_q(a, h, qf, U.qs);
    WaveStates<1> st;
    wave_attend<BF16, PS, 1>(a, h, qf, pg, st);
    fold_publish<1>(a, kStampMiss, pub_dst(a, h, a.n_spec), ep, st, 1u, U.attn);
  }
  update_window<J>(a, a.win + 4 * h, qn, key, cand, (9 * a.kextra_a) / 4, keep_window, U.sel.sel);
  if (a.late) update_window<J>(a, a.win + 4 * h + 2, qn, key, cand, kLateRank(a.kextra_a), true, U.sel.sel);
}

// Short candidate lists (at most 1024): wave 0 selects A, publishes the threshold and
// the list to attend, and writes the outputs, with no barrier; waves 1 and 2 meanwhile
// derive the next step's candidate bounds from the same list.
template <bool BF16, int PS>
__device__ __forceinline__ void select_wave(const FusedLaunch& a, uint32_t ep, int h, int total, float qn,
                                            const SelThreshold& th, int nM_done, FLds& U) {
  FSelLds& L = U.sel;
  constexpr int NK = kCandWave / kWave;
  const int t = threadIdx.x, lane = lane_id(), w = t / kWave;
  const bool prr = a.schedule == 1;
  uint32_t key[NK];
  int page[NK];
  uint64_t cand = 0, force = 0, lateb = 0, inP = 0;
  // unconditional LDS loads (slots past the list read stale words and are masked), so
  // that they issue back to back instead of one branch at a time
  static_assert(kCandWave <= kCandMax, "one-wave slots lie inside the LDS list");
  uint32_t pv[NK];
#pragma unroll
  for (int j = 0; j < NK; ++j) {
    key[j] = L.ck[j * kWave + lane];
    pv[j] = L.cpg[j * kWave + lane];
  }
  uint32_t pw[NK];
#pragma unroll
  for (int j = 0; j < NK; ++j) {
    const bool v = j * kWave + lane < total;
    key[j] = v ? key[j] : 0u;
    pv[j] = v ? pv[j] : 0u;
    page[j] = (int)(pv[j] & 0x3fffffffu);
    pw[j] = prr ? L.bitP[(page[j] >> 5) & (PRR_MAX_PAGES_DEV / 32 - 1)] : 0u;
  }
#pragma unroll
  for (int j = 0; j < NK; ++j) {
    const bool v = j * kWave + lane < total;
    if (v && (pv[j] >> 31)) force |= 1ull << j;
    if (v && !(pv[j] >> 31)) cand |= 1ull << j;
    if (v && ((pv[j] >> 30) & 1u)) lateb |= 1ull << j;
    if (v && ((pw[j] >> (page[j] & 31)) & 1u)) inP |= 1ull << j;
  }
  if (w == 0) {
    // the threshold was published already unless a tie at T is cut by page order
    const bool early = th.mode != 2 || th.need_eq >= th.eq_total;
    int eq_cut = kEqAll;
    const uint64_t inA = wsel_membership<NK>(key, page, cand, force, th, &eq_cut);
    if (prr && !early) {
      eq_cut = __builtin_amdgcn_readfirstlane(wave_umin((uint32_t)eq_cut));
      if (lane == 0) {
        publish_thr(a, h, th.T, (uint32_t)th.mode | ((uint32_t)eq_cut << 2), ep);
      }
    }
    // pages of late speculation: flagged, within the late capacity, never in P^t
    // (nM_done >= 0: the missed list was published by the whole workgroup already)
    uint64_t inLate = 0;
    int ltot = 0;
    if (a.late && nM_done < 0) {
      const int capl = a.n_late * a.chunk;
#pragma unroll
      for (int j = 0; j < NK; ++j) {
        const bool f = (lateb >> j) & 1ull;
        const uint64_t bm = __ballot(f);
        if (f && ltot + lanes_below(bm) < capl && !((inP >> j) & 1ull)) inLate |= 1ull << j;
        ltot += __popcll(bm);
      }
      if (lane == 0) put_rep(a.t_lcnt, h, 0, (uint32_t)min(ltot, capl), ep);
    }
    const int nMiss = prr ? wave_isum(__popcll(inA & ~inP)) : 0;
    int nM = nM_done;
    if (nM_done < 0) {
      const bool drop = prr && a.mode == PRR_RECOMPUTE_ON_MISS && nMiss > 0;
      const uint64_t inM = (prr && !drop) ? (inA & ~inP & ~inLate) : inA;
      const uint32_t mflags = drop ? kDropSpec : 0u;
      nM = min(wave_isum(__popcll(inM)), a.cap);
      uint64_t* ml = a.t_mlist + (size_t)h * a.cap;
      int pos = 0;
#pragma unroll
      for (int j = 0; j < NK; ++j) {
        const bool in = (inM >> j) & 1ull;
        const uint64_t bm = __ballot(in);
        const int q = pos + lanes_below(bm);
        if (in && q < a.cap) put_tag(&ml[q], (uint32_t)page[j], ep);
        pos += __popcll(bm);
      }
      // (the missed-page workgroups attend M even when it is short: this workgroup's
      // other waves are still deriving the next step's bounds)
      if (lane == 0) publish_mcnt(a, h, (uint32_t)nM | mflags, ep);
    }
    // the selected list (an output) and the counts
    int32_t* sel = a.selected + (size_t)h * a.cap;
    int na = 0;
#pragma unroll
    for (int j = 0; j < NK; ++j) {
      const bool in = (inA >> j) & 1ull;
      const uint64_t bm = __ballot(in);
      const int q = na + lanes_below(bm);
      if (in && q < a.cap) sel[q] = page[j];
      na += __popcll(bm);
    }
    const int nPA = prr ? wave_isum(__popcll(inP & inA)) : 0;
    if (lane == 0) {
      a.selected_count[h] = min(na, a.cap);
      if (a.missed_count) a.missed_count[h] = prr ? nMiss : nM;
      if (a.wasted_count) a.wasted_count[h] = prr ? L.npv - nPA : 0;
      if (a.covered_count) a.covered_count[h] = prr ? max(nMiss - nM, 0) : 0;  // (0 when M = A)
    }
  } else if (w == 1 || (w == 2 && a.late)) {
    // the next step's lower bounds: rank 2.25|A| (candidates of A) and 1.25|A| (late pages)
    const int k = w == 1 ? (9 * a.kextra_a) / 4 : kLateRank(a.kextra_a);
    const SelThreshold th = wsel_threshold<NK>(key, cand, max(k, 1), L.ws[w], true);
    if (lane == 0 && th.mode == 2 && qn > 0.0f) a.win[4 * h + (w == 1 ? 0 : 2)] = __float_as_uint(key_value(th.T) / qn);
  }
}

// The missed list M = A \ P \ (late-covered pages) (serial schedule: A) by the whole
// workgroup right after the threshold, when no tie at T is cut (membership is then
// key >= T); slot i = t + 512 j of the candidate list, two per thread.  Publishes M,
// its count and the number of late-covered pages; returns |M|.
__device__ __forceinline__ int miss_block(const FusedLaunch& a, uint32_t ep, int h, int total, const SelThreshold& th,
                                          const uint32_t (&k2)[2], FSelLds& L) {
  const int t = threadIdx.x;
  const bool prr = a.schedule == 1;
  const int capl = a.late ? a.n_late * a.chunk : 0;
  bool inA[2], late[2], inP[2];
  int pg[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int i = t + kFT * j;
    const uint32_t pv = L.cpg[i];
    const bool v = i < total;
    pg[j] = v ? (int)(pv & 0x3fffffffu) : 0;
    const bool forced = v && (pv >> 31);
    inA[j] = forced || (v && (th.mode == 1 || (th.mode == 2 && k2[j] >= th.T)));
    late[j] = v && a.late && ((pv >> 30) & 1u);
    inP[j] = prr && v && bit_of(L.bitP, pg[j]);
  }
  // late-covered: flagged, among the first capl flagged slots, not in P^t
  int tot_l;
  const int el = block_exclusive_scan<kFT>((int)late[0] | ((int)late[1] << 16), L.cnt[1], tot_l);
  const int l0 = tot_l & 0xffff;
  const int pl[2] = {el & 0xffff, l0 + (el >> 16)};
  bool mM[2], mA[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const bool cov = late[j] && pl[j] < capl && !inP[j];
    mA[j] = inA[j] && !inP[j];
    mM[j] = prr ? (mA[j] && !cov) : inA[j];
  }
  int tot_m;
  const int em = block_exclusive_scan<kFT>((int)mM[0] | ((int)mM[1] << 10) | (((int)mA[0] + (int)mA[1]) << 20),
                                          L.cnt[1], tot_m);
  const int nMiss = tot_m >> 20;
  const bool drop = prr && a.mode == PRR_RECOMPUTE_ON_MISS && nMiss > 0;
  int q[2] = {em & 0x3ff, (tot_m & 0x3ff) + ((em >> 10) & 0x3ff)};
  int nM = (tot_m & 0x3ff) + ((tot_m >> 10) & 0x3ff);
  if (drop) {  // the speculation is discarded: M = A
    int tot_a;
    const int ea = block_exclusive_scan<kFT>((int)inA[0] | ((int)inA[1] << 16), L.cnt[1], tot_a);
    mM[0] = inA[0];
    mM[1] = inA[1];
    q[0] = ea & 0xffff;
    q[1] = (tot_a & 0xffff) + (ea >> 16);
    nM = (tot_a & 0xffff) + (tot_a >> 16);
  }
  nM = min(nM, a.cap);
  uint64_t* ml = a.t_mlist + (size_t)h * a.cap;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    if (mM[j] && q[j] < a.cap) put_tag(&ml[q[j]], (uint32_t)pg[j], ep);
  }
  // (the missed-page workgroups attend M even when it is short: this workgroup goes on
  // to derive the next step's bounds)
  if (t == 0) {
    publish_mcnt(a, h, (uint32_t)nM | (drop ? kDropSpec : 0u), ep);
    if (a.late) put_rep(a.t_lcnt, h, 0, (uint32_t)min(l0 + (tot_l >> 16), capl), ep);
  }
  return nM;
}

template <bool BF16, int PS>
__device__ __forceinline__ void role_select(const FusedLaunch& a, uint32_t ep, int h, FLds& U) {
  FSelLds& L = U.sel;
  const int t = threadIdx.x;
  const int n = a.num_pages, nw = (n + 31) >> 5;
  // bitmaps of the forced pages (fallback) and of P^t (PRR), |P^t| in npv
  for (int i = t; i < nw; i += kFT) {
    L.forceb[i] = 0u;
    L.bitP[i] = 0u;
  }
  if (t == 0) {
    L.eq_cut = kEqAll;
    L.npv = 0;
  }
  // the bins of the one-wave selects, cleared while the candidates are awaited
  if (t < 3 * kWave) wsel_clear(L.ws[t / kWave]);
  __syncthreads();
  if (t == 0 && a.n_forced > 0) {
#pragma unroll
    for (int i = 0; i < PRR_MAX_FORCED; ++i) {
      if (i >= a.n_forced) break;
      atomicOr(&L.forceb[a.forced[i] >> 5], 1u << (a.forced[i] & 31));
    }
  }
  // P^t and q are loaded while the candidates are polled
  int pe[PRR_MAX_CAP_DEV / kFT];
  const int pc = a.schedule == 1 ? min(max(a.pred_cur_count[h], 0), a.cap) : 0;
#pragma unroll
  for (int r = 0; r < PRR_MAX_CAP_DEV / kFT; ++r) {
    const int i = t + r * kFT;
    pe[r] = i < pc ? a.pred_cur[(size_t)h * a.cap + i] : -1;
  }
  float qv[16];
  qbar_load<BF16>(a, h, qv);
  // both are ready long before the candidates: built first
  int nv = 0;
#pragma unroll
  for (int r = 0; r < PRR_MAX_CAP_DEV / kFT; ++r) {
    const int p = pe[r];
    if (p >= 0 && p < n) {
      atomicOr(&L.bitP[p >> 5], 1u << (p & 31));
      ++nv;
    }
  }
  nv = block_sum<kFT>(nv, L.cnt[1]);  // P^t holds no duplicates
  if (t == 0) L.npv = nv;
  const float qn = qbar_finish(a, qv, L.qb);
  const FCand c = cand_load<true>(a, ep, h, 0, L.off, L.tot, L.ck, L.cpg);  // (barriers inside)
  if (t == 0) stamp(a, kStampGathered);
  if (a.kextra_a <= c.total - c.nforced && c.total <= kCandWave) {
    // the threshold by the whole workgroup straight from the list (two keys per thread),
    // published at once when no tie at T needs cutting; the one-wave pass that follows
    // derives the sets and lists from it
    uint32_t k2[2];
    bool c2[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int i = t + kFT * j;  // < kCandWave <= 2 kFT
      k2[j] = L.ck[i];
      c2[j] = i < c.total && !(L.cpg[i] >> 31);
    }
    const SelThreshold th = bsel_threshold<kFT>(k2, c2, a.kextra_a, L.bsel);
    const bool early = th.mode != 2 || th.need_eq >= th.eq_total;
    if (a.schedule == 1 && t == 0 && early) {
      publish_thr(a, h, th.T, (uint32_t)th.mode | ((uint32_t)kEqAll << 2), ep);
    }
    const int nM = early ? miss_block(a, ep, h, c.total, th, k2, L) : -1;
    select_wave<BF16, PS>(a, ep, h, c.total, qn, th, nM, U);
  } else if (a.kextra_a <= c.total - c.nforced && c.total <= kCandMax) {
    // one instantiation per path keeps the kernel's code (and its instruction-cache
    // footprint) small: 4 candidate slots per thread, 16 page slots in the fallback
    uint32_t key[4];
    int page[4];
    uint64_t cand, force;
    uint64_t late_bits;
    cand_slots<4>(c.total, L.ck, L.cpg, key, page, cand, force, &late_bits);
    select_finish<BF16, PS, 4>(a, ep, h, key, page, cand, force, late_bits, true, qn, U);
  } else {
    uint32_t key[16];
    int page[16];
    uint64_t cand, force;
    full_gather<16>(a, ep, a.t_score + (size_t)h * a.max_pages, L.forceb, key, page, cand, force);
#pragma unroll
    for (int j = 0; j < 16; ++j) key[j] = score_key(__uint_as_float(key[j]));
    select_finish<BF16, PS, 16>(a, ep, h, key, page, cand, force, 0ull, false, qn, U);
  }
  if (t == 0) stamp(a, kStampSelectDone);
}

// The rank that sets the next step's candidate window of the prediction: 2.5 |P|, wider
// with a trend term (gamma > 0), whose keys move more from step to step (at gamma = 0.25,
// 2.5 |P| left 7 % of launches with too few or too many candidates, each falling back to
// all 8192 keys at ~8 us; 4 |P| leaves about 1 %).  At most 6 |P|, within the middle path.
__device__ __forceinline__ int pred_window_rank(const FusedLaunch& a) {
  return (int)((float)a.kextra_p * fminf(2.5f + 6.0f * a.gamma, 6.0f));
}

// ------------------------------------------------------------------------ predict

template <int J>
__device__ __forceinline__ void predict_finish(const FusedLaunch& a, uint32_t ep, int h, const uint32_t (&key)[J],
                                               const int (&page)[J], uint64_t cand, uint64_t force, bool keep_window,
                                               float qe, FSelLds& L) {
  const SelThreshold th = sel2_threshold<kFT, J>(key, cand, a.kextra_p, L.sel);
  const uint64_t in = sel2_compact<kFT, J>(key, page, cand, force, th, a.pred_nxt + (size_t)h * a.cap, a.cap,
                                           a.pred_nxt_count + h, &L.eq_cut, L.sel);
  // P^{t+1} as a bitmap too (the late-speculation filter of the next step)
  const int nw = (a.num_pages + 31) >> 5, nwmax = (a.max_pages + 31) >> 5;
  for (int i = threadIdx.x; i < nw; i += kFT) L.bitP[i] = 0u;
  __syncthreads();
#pragma unroll
  for (int j = 0; j < J; ++j)
    if ((in >> j) & 1ull) atomicOr(&L.bitP[page[j] >> 5], 1u << (page[j] & 31));
  __syncthreads();
  for (int i = threadIdx.x; i < nw; i += kFT) a.pbits_nxt[(size_t)h * nwmax + i] = L.bitP[i];
  update_window<J>(a, a.win + 4 * h + 1, qe, key, cand, pred_window_rank(a), keep_window, L.sel);
}

// The next prediction from a short candidate list and the workgroup's threshold, as
// select_wave does for A: wave 0 writes P^{t+1} in page order, wave 1 finds the next
// step's bound of the candidates (rank 2.5 |P|), the other waves clear the bitmap meanwhile.
__device__ __forceinline__ void predict_wave(const FusedLaunch& a, int h, int total, float qe, const SelThreshold& th,
                                             FSelLds& L) {
  constexpr int NK = kCandWave / kWave;
  const int t = threadIdx.x, lane = lane_id(), w = t / kWave;
  const int nw = (a.num_pages + 31) >> 5, nwmax = (a.max_pages + 31) >> 5;
  uint32_t key[NK], pv[NK];
  int page[NK];
  uint64_t cand = 0, force = 0, in = 0;
  if (w < 2) {
#pragma unroll
    for (int j = 0; j < NK; ++j) {
      key[j] = L.ck[j * kWave + lane];
      pv[j] = L.cpg[j * kWave + lane];
    }
#pragma unroll
    for (int j = 0; j < NK; ++j) {
      const bool v = j * kWave + lane < total;
      key[j] = v ? key[j] : 0u;
      page[j] = v ? (int)(pv[j] & 0x3fffffffu) : 0;
      if (v && (pv[j] >> 31)) force |= 1ull << j;
      if (v && !(pv[j] >> 31)) cand |= 1ull << j;
    }
  }
  if (w == 0) {
    int eq_cut = kEqAll;
    in = wsel_membership<NK>(key, page, cand, force, th, &eq_cut);
    int32_t* out = a.pred_nxt + (size_t)h * a.cap;
    int n = 0;
#pragma unroll
    for (int j = 0; j < NK; ++j) {
      const bool m = (in >> j) & 1ull;
      const uint64_t bm = __ballot(m);
      const int q = n + lanes_below(bm);
      if (m && q < a.cap) out[q] = page[j];
      n += __popcll(bm);
    }
    if (lane == 0) a.pred_nxt_count[h] = min(n, a.cap);
  } else if (w == 1) {
    const SelThreshold th = wsel_threshold<NK>(key, cand, max(pred_window_rank(a), 1), L.ws[1], true);
    if (lane == 0 && th.mode == 2 && qe > 0.0f) a.win[4 * h + 1] = __float_as_uint(key_value(th.T) / qe);
  } else {
    for (int i = t - 2 * kWave; i < nw; i += kFT - 2 * kWave) L.bitP[i] = 0u;
  }
  __syncthreads();
  // P^{t+1} as a bitmap too (the late-speculation filter of the next step)
  if (w == 0) {
#pragma unroll
    for (int j = 0; j < NK; ++j)
      if ((in >> j) & 1ull) atomicOr(&L.bitP[page[j] >> 5], 1u << (page[j] & 31));
  }
  __syncthreads();
  for (int i = t; i < nw; i += kFT) a.pbits_nxt[(size_t)h * nwmax + i] = L.bitP[i];
}

template <bool BF16>
__device__ __forceinline__ void role_predict(const FusedLaunch& a, uint32_t ep, int h, FLds& U) {
  FSelLds& L = U.sel;
  const int t = threadIdx.x;
  const int n = a.num_pages, nw = (n + 31) >> 5;
  for (int i = t; i < nw; i += kFT) L.forceb[i] = 0u;
  // the bins of the one-wave selects, cleared while the candidates are awaited
  if (t < 2 * kWave) wsel_clear(L.ws[t / kWave]);
  __syncthreads();
  if (t == 0 && a.n_forced > 0) {
#pragma unroll
    for (int i = 0; i < PRR_MAX_FORCED; ++i) {
      if (i >= a.n_forced) break;
      atomicOr(&L.forceb[a.forced[i] >> 5], 1u << (a.forced[i] & 31));
    }
  }
  const float qe0 = __uint_as_float(a.win[4 * h + 3]);  // read before any score workgroup ends
  float qv[16];
  qbar_load<BF16>(a, h, qv);
  const float qe = qn_ema(a, qbar_finish(a, qv, L.qb), qe0);
  const FCand c = cand_load<false>(a, ep, h, 1, L.off, L.tot, L.ck, L.cpg);  // (no hurry: the next step's set)
  if (t == 0) stamp(a, kStampGathered);
  // every score workgroup has read the bounds: the scale of the next step's keys
  if (t == 0) a.win[4 * h + 3] = __float_as_uint(qe);
  if (a.kextra_p <= c.total - c.nforced && c.total <= kCandWave) {
    // the threshold of P^{t+1} by the whole workgroup (two keys per thread); then one wave
    // writes the list while another finds the next step's bound
    uint32_t k2[2];
    bool c2[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int i = t + kFT * j;  // < kCandWave <= 2 kFT
      k2[j] = L.ck[i];
      c2[j] = i < c.total && !(L.cpg[i] >> 31);
    }
    const SelThreshold th = bsel_threshold<kFT>(k2, c2, a.kextra_p, L.bsel);
    if (t == 0) stamp(a, kStampThreshold);
    predict_wave(a, h, c.total, qe, th, L);
  } else if (a.kextra_p <= c.total - c.nforced && c.total <= kCandMax) {
    if (t == 0) stamp(a, kStampMissed);  // (predict workgroups: the middle path was taken)
    uint32_t key[4];
    int page[4];
    uint64_t cand, force;
    cand_slots<4>(c.total, L.ck, L.cpg, key, page, cand, force, nullptr);
    predict_finish<4>(a, ep, h, key, page, cand, force, true, qe, L);
  } else {
    if (t == 0) stamp(a, kStampSelectDone);  // (predict workgroups: the full gather was taken)
    uint32_t key[16];
    int page[16];
    uint64_t cand, force;
    full_gather<16>(a, ep, a.t_pkey + (size_t)h * a.max_pages, L.forceb, key, page, cand, force);
    predict_finish<16>(a, ep, h, key, page, cand, force, false, qe, L);
  }
  if (t == 0) stamp(a, kStampPredictDone);
}

// ------------------------------------------------------------------------ spec / miss

// Membership of this wave's pages in A, from their scores and the published threshold
// (all loads issued together, then waited for); returns `keep` without the pages not in A.
// Called by every wave of the workgroup (it holds a barrier).
template <int NPW>
__device__ __forceinline__ uint32_t keep_in_A(const FusedLaunch& a, uint32_t ep, int h, const int (&pg)[NPW], uint32_t keep,
                                              uint32_t* bc) {
  const uint64_t* ts = a.t_score + (size_t)h * a.max_pages;
  uint64_t vs[NPW];
#pragma unroll
  for (int k = 0; k < NPW; ++k) vs[k] = keep ? get_tag(&ts[max(pg[k], 0)]) : 0ull;
  if (threadIdx.x < kWave) {
    const uint64_t* thr = rep_at(a.t_thr, h, blockIdx.x);
    uint64_t v0 = 0, v1 = 0;
    for (int it = 0; it < kFSpin; ++it) {
      v0 = get_tag(thr);
      v1 = get_tag(thr + 1);
      if (tag_is(v0, ep) && tag_is(v1, ep)) break;
      __builtin_amdgcn_s_sleep(2);
      if (it == kFSpin - 1 && threadIdx.x == 0) atomicOr(a.flags, kFlagSpinTimeout);
    }
    if (threadIdx.x == 0) {
      bc[0] = (uint32_t)v0;
      bc[1] = (uint32_t)v1;
    }
  }
  __syncthreads();
  if (!keep) return keep;
  // the scores were published before the threshold; one that is not visible yet is
  // awaited (the rare case, kept out of the common path's instruction stream)
  bool stale = false;
#pragma unroll
  for (int k = 0; k < NPW; ++k) stale = stale || (pg[k] >= 0 && !tag_is(vs[k], ep));
  if (__builtin_expect(stale, 0)) {
#pragma unroll
    for (int k = 0; k < NPW; ++k)
      if (pg[k] >= 0) vs[k] = tagged(vs[k], &ts[pg[k]], ep, a.flags);
  }
  uint32_t sc[NPW];
#pragma unroll
  for (int k = 0; k < NPW; ++k) sc[k] = (uint32_t)vs[k];
  const uint32_t T = bc[0];
  const uint32_t me = bc[1];
  const int mode = (int)(me & 3u), eq_cut = (int)(me >> 2);
#pragma unroll
  for (int k = 0; k < NPW; ++k) {
    if (pg[k] < 0 || page_forced(a, pg[k])) continue;
    const uint32_t key = score_key(__uint_as_float(sc[k]));
    const bool in = mode == 1 || (mode == 2 && (key > T || (key == T && pg[k] <= eq_cut)));
    if (!in) keep &= ~(1u << k);
  }
  return keep;
}

// One page per wave: the page states go to LDS before A is known; once the threshold is
// published, wave 0 decides for the eight pages which are in A (so one barrier follows
// the threshold instead of two), and the kept states are combined and published.
__device__ __forceinline__ void keep_fold_publish(const FusedLaunch& a, int slot, uint32_t ep, int h, int pg,
                                                  WaveStates<1>& st, const PubDst& pd, FAttnLds& L) {
  const int t = threadIdx.x, lane = lane_id(), w = t / kWave;
  fold_write<1>(st, 1u, L);
  if (lane == 0) L.kpg[w] = pg;
  __syncthreads();
  if (w == 0) {
    const int p = lane < kFW ? L.kpg[lane] : -1;
    const uint64_t* ts = a.t_score + (size_t)h * a.max_pages;
    // the page's score is polled with the threshold (it was published before it)
    const uint64_t* sp = &ts[max(p, 0)];
    const uint64_t* thr = rep_at(a.t_thr, h, blockIdx.x);
    uint64_t v0 = 0, v1 = 0, vs = 0;
    for (int it = 0; it < kFSpin; ++it) {
      v0 = get_tag(thr);
      v1 = get_tag(thr + 1);
      vs = get_tag(sp);
      if (__ballot(!tag_is(v0, ep) || !tag_is(v1, ep) || (p >= 0 && !tag_is(vs, ep))) == 0ull) break;
      __builtin_amdgcn_s_sleep(2);
      if (it == kFSpin - 1 && lane == 0) atomicOr(a.flags, kFlagSpinTimeout);
    }
    const uint32_t sc = p >= 0 ? (uint32_t)vs : 0u;
    const uint32_t T = (uint32_t)v0, me = (uint32_t)v1;
    const int mode = (int)(me & 3u), eq_cut = (int)(me >> 2);
    const uint32_t key = score_key(__uint_as_float(sc));
    const bool in = p >= 0 && (page_forced(a, p) || mode == 1 || (mode == 2 && (key > T || (key == T && p <= eq_cut))));
    const uint32_t m = (uint32_t)__ballot(in) & ((1u << kFW) - 1u);
    if (lane == 0) L.kmask = m;
  }
  __syncthreads();
  combine_publish(a, slot, pd, ep, L.kmask, L);
}

template <bool BF16, int PS, int NPW>
__device__ __forceinline__ void role_spec(const FusedLaunch& a, uint32_t ep, int h, int c, FLds& U) {
  const int count = min(max(a.pred_cur_count[h], 0), a.cap);
  const int start = c * a.chunk;
  if (start >= count) return;
  const int cnt = min(a.chunk, count - start);
  const int w = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
  u32x4_t qf[4];
  load_q(a, h, qf, U.qs);
  int pg[NPW];
  uint32_t keep = 0;
#pragma unroll
  for (int k = 0; k < NPW; ++k) {
    const int i = w + kFW * k;
    int p = i < cnt ? a.pred_cur[(size_t)h * a.cap + start + i] : -1;
    p = __builtin_amdgcn_readfirstlane(p);
    if (i < cnt && (p < 0 || p >= a.num_pages)) {
      if (lane_id() == 0) atomicOr(a.flags, kFlagBadListEntry);
      p = -1;
    }
    pg[k] = p;
    if (p >= 0) keep |= 1u << k;
  }
  WaveStates<NPW> st;
  wave_attend<BF16, PS, NPW>(a, h, qf, pg, st);
  if (threadIdx.x == 0) stamp(a, kStampAttended);
  const PubDst pd = pub_dst(a, h, c);
  if constexpr (NPW == 1) {
    if (a.mode != PRR_KEEP_WASTED) {
      keep_fold_publish(a, kStampSpec, ep, h, pg[0], st, pd, U.attn);
      return;
    }
  } else {
    if (a.mode != PRR_KEEP_WASTED) keep = keep_in_A<NPW>(a, ep, h, pg, keep, U.bc);
  }
  fold_publish<NPW>(a, kStampSpec, pd, ep, st, keep, U.attn);
}

// Late speculation (PRR schedule): as soon as this step's scores exist, the pages just
// above the selection threshold that P^t missed (listed by the score workgroups) are
// attended, one state per page; once A is known the states of pages in A are folded.
template <bool BF16, int PS, int NPW>
__device__ __forceinline__ void role_late(const FusedLaunch& a, uint32_t ep, int h, int u, FLds& U) {
  FSelLds& L = U.sel;
  const int t = threadIdx.x;
  const int w = __builtin_amdgcn_readfirstlane((int)(t / kWave));
  u32x4_t qf[4];
  load_q(a, h, qf, U.qs);
  // P^t as an LDS bitmap: a page of P^t is never attended here (the hint bitmap the
  // score workgroups filtered with may be stale)
  const int n = a.num_pages, nw = (n + 31) >> 5;
  for (int i = t; i < nw; i += kFT) L.bitP[i] = 0u;
  int pe[PRR_MAX_CAP_DEV / kFT];
  const int pc = min(max(a.pred_cur_count[h], 0), a.cap);
#pragma unroll
  for (int r = 0; r < PRR_MAX_CAP_DEV / kFT; ++r) {
    const int i = t + r * kFT;
    pe[r] = i < pc ? a.pred_cur[(size_t)h * a.cap + i] : -1;
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < PRR_MAX_CAP_DEV / kFT; ++r)
    if (pe[r] >= 0 && pe[r] < n) atomicOr(&L.bitP[pe[r] >> 5], 1u << (pe[r] & 31));
  const FCand c = cand_load<false>(a, ep, h, 2, L.off, L.tot, L.ck, L.cpg);  // (barriers inside)
  // More late pages than one list in LDS holds (after the candidate windows were reset):
  // the list was not loaded.  The candidates of A are then at least as many, so the select
  // workgroup takes its fallback over all scores and publishes a late count of 0, and the
  // merge reads no late state.
  if (c.total > kCandMax) return;
  if (t == 0) stamp(a, kStampLateList);
  const int cover = min(c.total, a.n_late * a.chunk);
  const int start = u * a.chunk;
  if (start >= cover) return;
  const int cnt = min(a.chunk, cover - start);
  int pg[NPW], ph[NPW];
  uint32_t keep = 0;
#pragma unroll
  for (int k = 0; k < NPW; ++k) {
    const int i = w + kFW * k;
    int p = -1, q = -1;
    if (i < cnt) {
      p = (int)(L.cpg[start + i] & 0x3fffffffu);
      q = (int)L.ck[start + i];  // its physical page
      if (p >= n || bit_of(L.bitP, p)) p = -1;
    }
    pg[k] = __builtin_amdgcn_readfirstlane(p);
    ph[k] = __builtin_amdgcn_readfirstlane(p >= 0 ? q : -1);
    if (pg[k] >= 0) keep |= 1u << k;
  }
  __syncthreads();  // the list is read before the attention reuses the LDS
  WaveStates<NPW> st;
  wave_attend<BF16, PS, NPW>(a, h, qf, pg, st, ph);
  if (t == 0) stamp(a, kStampAttended);
  const PubDst pd = pub_dst(a, h, a.n_spec + a.n_miss + u);
  if constexpr (NPW == 1) {
    keep_fold_publish(a, kStampLate, ep, h, pg[0], st, pd, U.attn);
  } else {
    keep = keep_in_A<NPW>(a, ep, h, pg, keep, U.bc);
    fold_publish<NPW>(a, kStampLate, pd, ep, st, keep, U.attn);
  }
}

// Chunk c of the missed list (its state to slot n_spec + c); false once the list holds no
// chunk c.  The count and the chunk's entries are loaded together; the entries are
// published before the count, so they are usually valid when the count is.
template <bool BF16, int PS, int NPW>
__device__ __forceinline__ bool miss_chunk(const FusedLaunch& a, uint32_t ep, int h, int c, bool first, FLds& U) {
  const int start = c * a.chunk;
  const int w = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
  u32x4_t qf[4];  // (q is staged once; a later chunk reads it from LDS again)
  if (first) load_q(a, h, qf, U.qs);
  else fetch_q(a, qf, U.qs);
  static_assert(1 + kFW * NPW <= 2 + 2 * kFW, "broadcast area");
  const uint64_t* ml = a.t_mlist + (size_t)h * a.cap;
  if (w == 0) {
    // lane l < kFW * NPW polls entry start + l (page k of wave w is entry w + kFW k)
    const int lane = lane_id();
    const int i = start + lane;
    uint64_t vm = 0, ve = 0;
    for (int it = 0; it < kFSpin; ++it) {
      vm = get_tag(rep_at(a.t_mcnt, h, c));
      if (lane < kFW * NPW) ve = get_tag(&ml[min(i, a.cap - 1)]);  // (only the entries of this chunk)
      if (tag_is(vm, ep)) {
        const uint32_t mv = (uint32_t)vm;
        const int nm = (mv & kSelfMiss) ? 0 : (int)(mv & kCountMask);
        if (__ballot(lane < kFW * NPW && i < nm && !tag_is(ve, ep)) == 0ull) break;
      }
      __builtin_amdgcn_s_sleep(2);
      if (it == kFSpin - 1 && lane == 0) atomicOr(a.flags, kFlagSpinTimeout);
    }
    if (lane == 0) U.bc[0] = (uint32_t)vm;
    if (lane < kFW * NPW) U.bc[1 + lane] = (uint32_t)ve;
  }
  __syncthreads();  // (a previous chunk's readers of U.bc are past its publishing barrier)
  const uint32_t mv = U.bc[0];
  if (mv & kSelfMiss) return false;
  const int nM = (int)(mv & kCountMask);
  if (start >= nM) return false;
  const int cnt = min(a.chunk, nM - start);
  int pg[NPW];
  uint32_t keep = 0;
#pragma unroll
  for (int k = 0; k < NPW; ++k) {
    const int i = w + kFW * k;
    int p = i < cnt ? (int)U.bc[1 + i] : -1;
    p = __builtin_amdgcn_readfirstlane(p);
    if (i < cnt && (p < 0 || p >= a.num_pages)) {  // only after a timed-out wait
      if (lane_id() == 0) atomicOr(a.flags, kFlagBadListEntry);
      p = -1;
    }
    pg[k] = p;
    if (p >= 0) keep |= 1u << k;
  }
  WaveStates<NPW> st;
  wave_attend<BF16, PS, NPW>(a, h, qf, pg, st);
  fold_publish<NPW>(a, kStampMiss, pub_dst(a, h, a.n_spec + c), ep, st, keep, U.attn);
  return true;
}

// Missed-list workgroup u of a KV head: chunks u, u + miss_wgs, .. (one pass when the list
// is short, as it is once late speculation covers most of A).  Instances of two pages per
// wave take one chunk each (the launcher gives them a workgroup per chunk): a loop around
// their attention would cost them occupancy.
template <bool BF16, int PS, int NPW>
__device__ __forceinline__ void role_miss(const FusedLaunch& a, uint32_t ep, int h, int u, FLds& U) {
  if constexpr (NPW == 1) {
    for (int c = u; c < a.n_miss; c += a.miss_wgs)
      if (!miss_chunk<BF16, PS, NPW>(a, ep, h, c, c == u, U)) return;
  } else {
    miss_chunk<BF16, PS, NPW>(a, ep, h, u, true, U);
  }
}

// ------------------------------------------------------------------------ merge

template <bool BF16>
__device__ __forceinline__ void role_merge(const FusedLaunch& a, uint32_t ep, int h, int qn, FMergeLds& L, uint32_t* bc) {
  const float kNegInf = -__builtin_inff();
  const int t = threadIdx.x, lane = lane_id(), w = t / kWave;
  const int G = a.group, C = a.chunk;
  int nspec = 0;
  if (a.schedule == 1) nspec = (min(max(a.pred_cur_count[h], 0), a.cap) + C - 1) / C;
  if (t < kWave) {
    uint64_t v0 = 0, v1 = 0;
    for (int it = 0; it < kFSpin; ++it) {
      v0 = get_tag(rep_at(a.t_mcnt, h, qn));
      v1 = a.late ? get_tag(rep_at(a.t_lcnt, h, qn)) : ((uint64_t)ep << 32);
      if (tag_is(v0, ep) && tag_is(v1, ep)) break;
      __builtin_amdgcn_s_sleep(2);
      if (it == kFSpin - 1 && t == 0) atomicOr(a.flags, kFlagSpinTimeout);
    }
    if (t == 0) {
      bc[0] = (uint32_t)v0;
      bc[1] = (uint32_t)v1;
    }
  }
  __syncthreads();
  const uint32_t mv = bc[0];
  const int nM = (int)(mv & kCountMask);
  const int nmiss = (mv & kSelfMiss) ? 1 : (nM + C - 1) / C;
  if (mv & kDropSpec) nspec = 0;
  const int nlate = a.late ? ((int)bc[1] + C - 1) / C : 0;
  const int total = nspec + nmiss + nlate;
  // state i lives in slot i (speculation chunks), n_spec + (i - nspec) (missed chunks) or
  // n_spec + n_miss + (i - nspec - nmiss) (late-speculation chunks)
  const uint64_t* pml = a.t_part + ((size_t)h * a.nparts * G + qn) * 2;
  const float* po = a.part_o + ((size_t)h * a.nparts * G + qn) * kHeadDim;
  const int gap1 = a.n_spec - nspec, gap2 = a.n_spec + a.n_miss - nspec - nmiss;
#define PRR_SLOT(i) ((size_t)((i) < nspec ? (i) : ((i) < nspec + nmiss ? (i) + gap1 : (i) + gap2)) * G)

  // Wave w merges states w, w + 8, .. on its own (no barrier until the end): lane k polls
  // the (m, l) of state w + 8k (the outputs of a state are complete once its (m, l) are
  // current), then the wave loads the outputs of its states, lane l columns 2l and 2l + 1,
  // and folds them in state order into a running (max, sum, output).
  float Mw = kNegInf, Lw = 0.0f, ax = 0.0f, ay = 0.0f;
  const int nk = total > w ? (total - w + kFW - 1) / kFW : 0;
  for (int k0 = 0; k0 < nk; k0 += kWave) {
    const int k = k0 + lane;
    const bool mine = k < nk;
    const uint64_t* p = pml + PRR_SLOT(w + kFW * min(k, nk - 1)) * 2;
    uint64_t vm = 0, vl = 0;
    for (int it = 0; it < kFSpin; ++it) {
      vm = get_tag(p);
      vl = get_tag(p + 1);
      if (__ballot(mine && !(tag_is(vm, ep) && tag_is(vl, ep))) == 0ull) break;
      __builtin_amdgcn_s_sleep(2);
      if (it == kFSpin - 1 && lane == 0) atomicOr(a.flags, kFlagSpinTimeout);
    }
    const float li = mine ? __uint_as_float((uint32_t)vl) : 0.0f;
    const float mi = li > 0.0f ? __uint_as_float((uint32_t)vm) : kNegInf;
    const float Mn = fmaxf(Mw, wave_max(mi));
    if (Mn == kNegInf) continue;  // no state of this batch holds anything
    const float sc = Lw > 0.0f ? exp2f((Mw - Mn) * kLog2e) : 0.0f;
    ax *= sc;
    ay *= sc;
    const float wi = li > 0.0f ? li * exp2f((mi - Mn) * kLog2e) : 0.0f;
    Lw = Lw * sc + wave_sum(wi);
    Mw = Mn;
    const int nb = min(kWave, nk - k0);
    constexpr int kB = 8;
    for (int b0 = 0; b0 < nb; b0 += kB) {
      uint64_t ov[kB];
#pragma unroll
      for (int r = 0; r < kB; ++r) {
        const int i = w + kFW * (k0 + min(b0 + r, nb - 1));
        ov[r] = __hip_atomic_load(reinterpret_cast<uint64_t*>(const_cast<float*>(po + PRR_SLOT(i) * kHeadDim)) + lane,
                                  __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
#pragma unroll
      for (int r = 0; r < kB; ++r) {
        const float wr = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wi), min(b0 + r, kWave - 1)));
        const float wgt = b0 + r < nb ? wr : 0.0f;
        ax += wgt * __uint_as_float((uint32_t)ov[r]);
        ay += wgt * __uint_as_float((uint32_t)(ov[r] >> 32));
      }
    }
  }
  *reinterpret_cast<float2*>(&L.acc[w][2 * lane]) = make_float2(ax, ay);
  if (lane == 0) {
    L.red[0][w] = Mw;
    L.red[1][w] = Lw;
  }
  __syncthreads();
  if (t < kHeadDim) {
    const int c = t;
    float M = kNegInf;
#pragma unroll
    for (int ww = 0; ww < kFW; ++ww)
      if (L.red[1][ww] > 0.0f) M = fmaxf(M, L.red[0][ww]);
    float Lsum = 0.0f, sum = 0.0f;
#pragma unroll
    for (int ww = 0; ww < kFW; ++ww) {
      const float lw = L.red[1][ww];
      const float f = lw > 0.0f ? exp2f((L.red[0][ww] - M) * kLog2e) : 0.0f;
      Lsum += lw * f;
      sum += L.acc[ww][c] * f;
    }
    const float o = Lsum > 0.0f ? sum / Lsum : 0.0f;
    const size_t row = (size_t)h * G + qn;
    a.out_o32[row * kHeadDim + c] = o;
    if (a.out_o) static_cast<uint16_t*>(a.out_o)[row * kHeadDim + c] = (uint16_t)f2h_rne<BF16>(o);
    if (c == 0) {
      a.out_m[row] = Lsum > 0.0f ? M : kNegInf;
      a.out_l[row] = Lsum;
      stamp(a, kStampMerge);
    }
  }
#undef PRR_SLOT
}

// ------------------------------------------------------------------------ kernel

template <bool BF16, int PS, int NPW>
__device__ __forceinline__ void fused_roles(const FusedLaunch& a, uint32_t ep, FLds& U) {
  int b = blockIdx.x;
  const int H = a.num_kv_heads;
  if (b < H * a.n_score) {
    role_score<BF16, PS>(a, ep, b / a.n_score, b % a.n_score, U.score);
    return;
  }
  b -= H * a.n_score;
  if (b < H) {
    role_select<BF16, PS>(a, ep, b, U);
    return;
  }
  b -= H;
  if (a.schedule != 0) {
    if (b < H) {
      role_predict<BF16>(a, ep, b, U);
      return;
    }
    b -= H;
  }
  if (a.schedule == 2) return;
  if (a.schedule == 1) {
    if (b < H * a.n_spec) {
      role_spec<BF16, PS, NPW>(a, ep, b / a.n_spec, b % a.n_spec, U);
      return;
    }
    b -= H * a.n_spec;
    if (b < H * a.n_late) {
      role_late<BF16, PS, NPW>(a, ep, b / a.n_late, b % a.n_late, U);
      return;
    }
    b -= H * a.n_late;
  }
  if (b < H * a.miss_wgs) {
    role_miss<BF16, PS, NPW>(a, ep, b / a.miss_wgs, b % a.miss_wgs, U);
    return;
  }
  b -= H * a.miss_wgs;
  if (b < H * a.group) role_merge<BF16>(a, ep, b / a.group, b % a.group, U.merge, U.bc);
}

template <bool BF16, int PS, int NPW>
__global__ __launch_bounds__(kFT) void fused_step_kernel(const FusedLaunch a) {
  __shared__ FLds U;
  if (threadIdx.x == 0) stamp(a, kStampStart);
  // the epoch of this call: the kernel argument, or a device word that the caller
  // advances between replays of a captured launch (written by an earlier launch, so
  // visible at this launch's start)
  const uint32_t ep = a.epoch_dev ? *a.epoch_dev : a.epoch;
  fused_roles<BF16, PS, NPW>(a, ep, U);
  // the end of the workgroup's last wave (waves of a role may finish at different times)
  if (a.stamps && (threadIdx.x & (kWave - 1)) == 0)
    atomicMax(&a.stamps[(size_t)kStampEnd * kStampMaxWorkgroups + blockIdx.x],
              (unsigned long long)__builtin_amdgcn_s_memrealtime());
}

}  // namespace

// One instance of the fused kernel, launched on `grid` workgroups.  Instances are spread
// over several translation units (explicit instantiations below each include of this
// file), so that they compile in parallel.
//
// The late read-ahead keeps a score workgroup resident until its loads return.  It is
// used only when the whole grid is resident at once: otherwise the workgroups dispatched
// last (late, missed-page and merge roles) wait for those slots.
// Workgroups of this instance resident at once on the current device (cached per device),
// or 0 when the runtime cannot tell.
template <bool BF16, int PS, int NPW>
int resident_inst() {
  constexpr int kMaxDevices = 64;
  static int resident[kMaxDevices];  // (0 = not known yet)
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  int cap = dev >= 0 && dev < kMaxDevices ? resident[dev] : 0;
  if (cap == 0) {
    int per_cu = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(fused_step_kernel<BF16, PS, NPW>),
                                                     kFT, 0) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      return 0;
    cap = per_cu * cus;
    if (dev >= 0 && dev < kMaxDevices) resident[dev] = cap;
  }
  return cap;
}

template <bool BF16, int PS, int NPW>
hipError_t launch_fused_inst(int grid, const FusedLaunch& a, hipStream_t stream) {
  const int cap = resident_inst<BF16, PS, NPW>();
  FusedLaunch b = a;
  b.readahead = a.readahead && grid <= cap;
  void* args[] = {&b};
  return hipLaunchKernel(reinterpret_cast<const void*>(fused_step_kernel<BF16, PS, NPW>), dim3(grid), dim3(kFT), args,
                         0, stream);
}

}  // namespace prr
