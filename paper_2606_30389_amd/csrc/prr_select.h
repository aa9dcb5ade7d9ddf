// Block-wide exact top-K over keys held in registers (the selection of Section 2.1 /
// Appendix A.1 and the predicted-set selection of Section 4.1): NT threads, J keys per
// thread, thread t (wave w, lane) owning pages w*J*64 + j*64 + lane, so that the
// pages of a wave are contiguous and (w, j, lane) is ascending page order.
//
// The threshold key T (the kextra-th largest candidate key) is found by radix passes
// over 2048 LDS bins spanning the current key range [lo, hi]: LDS atomics build the
// histogram, one wave scans it from the top (32 bins per lane, DPP prefix sum) and
// every pass keeps only the bin that holds the wanted rank.  As soon as that bin holds
// at most 64 keys they are ranked directly by one wave instead of another pass, so a
// select usually takes one histogram pass.  Ties at T are broken by page index: the
// first need_eq keys equal to T in page order are taken.
#pragma once

#include "prr_device.h"

namespace prr {

constexpr int kSel2Log2Bins = 11;
constexpr int kSel2Bins = 1 << kSel2Log2Bins;
constexpr int kSel2Small = 64;

struct Sel2Lds {
  uint32_t hist[2][kSel2Bins];
  uint32_t small[kSel2Small];
  int nsmall;
  int red[3][16];
  int res[8];
};

struct SelThreshold {
  int mode;       // 0: no candidate taken, 1: every candidate, 2: candidates above T and ties
  uint32_t T;
  int need_eq;    // keys equal to T to take, in page order
  int eq_total;   // keys equal to T among the candidates
};

__host__ __device__ inline int sel2_j(int n, int nt) {
  int j = 1;
  while (j * nt < n) j <<= 1;
  return j;
}

template <int J>
__device__ __forceinline__ int sel2_page(int j) {
  return (threadIdx.x / kWave) * J * kWave + j * kWave + lane_id();
}

template <int NT, int J>
__device__ __forceinline__ SelThreshold sel2_threshold(const uint32_t (&key)[J], uint64_t cand, int kextra, Sel2Lds& S) {
  static_assert(NT >= 128 && NT <= 1024 && NT % kWave == 0, "block size");
  static_assert(J >= 1 && J <= 64, "keys per thread");
  constexpr int NW = NT / kWave;
  const int t = threadIdx.x, lane = lane_id(), w = t / kWave;

  int cnt = __popcll(cand);
  uint32_t lo = 0xffffffffu, hi = 0u;
#pragma unroll
  for (int j = 0; j < J; ++j) {
    if ((cand >> j) & 1ull) {
      lo = min(lo, key[j]);
      hi = max(hi, key[j]);
    }
  }
  cnt = wave_isum(cnt);
  lo = wave_umin(lo);
  hi = wave_umax(hi);
  for (int b = t; b < kSel2Bins / 4; b += NT) reinterpret_cast<uint4*>(S.hist[0])[b] = make_uint4(0, 0, 0, 0);
  if (t == 0) S.nsmall = 0;
  if (lane == 0) {
    S.red[0][w] = cnt;
    S.red[1][w] = (int)lo;
    S.red[2][w] = (int)hi;
  }
  __syncthreads();
  cnt = 0;
  lo = 0xffffffffu;
  hi = 0u;
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    cnt += S.red[0][i];
    lo = min(lo, (uint32_t)S.red[1][i]);
    hi = max(hi, (uint32_t)S.red[2][i]);
  }

  SelThreshold r;
  r.mode = 0;
  r.T = 0;
  r.need_eq = 0;
  r.eq_total = 0;
  if (kextra <= 0 || cnt == 0) return r;
  if (kextra >= cnt) {
    r.mode = 1;
    return r;
  }
  r.mode = 2;
  int rank = kextra;  // 1 = largest, among the candidate keys in [lo, hi]
  int inrange = cnt;
  int buf = 0;
  r.T = lo;
  r.need_eq = rank;
  r.eq_total = inrange;
  for (int pass = 0; pass < 3; ++pass) {
    const uint32_t range = hi - lo;
    if (range == 0) {
      r.T = lo;
      r.need_eq = rank;
      r.eq_total = inrange;
      break;
    }
    const int bits = 32 - __clz(range);
    const int shift = bits > kSel2Log2Bins ? bits - kSel2Log2Bins : 0;
    uint32_t* hist = S.hist[buf];
#pragma unroll
    for (int j = 0; j < J; ++j) {
      if (((cand >> j) & 1ull) && key[j] >= lo && key[j] <= hi) atomicAdd(&hist[(key[j] - lo) >> shift], 1u);
    }
    __syncthreads();
    if (w == 0) {
      // lane l owns bins [2048 - 32(l+1), 2048 - 32l), summed, then a prefix over lanes
      // (lane 0 holds the top bins) finds the lane holding rank `rank`; its 32 bins are
      // then spread over lanes 0..31 and a second prefix finds the bin
      const int base = kSel2Bins - 32 * (lane + 1);
      const uint4* hb = reinterpret_cast<const uint4*>(hist + base);
      int s = 0;
#pragma unroll
      for (int v = 0; v < 8; ++v) {
        const uint4 x = hb[v];
        s += (int)(x.x + x.y + x.z + x.w);
      }
      const int incl = wave_inclusive_scan(s);
      const int excl = incl - s;
      const uint64_t hit = __ballot(excl < rank && rank <= incl);
      const int ls = __builtin_amdgcn_readfirstlane(__ffsll((long long)hit) - 1);
      const int ex = __builtin_amdgcn_readlane(excl, ls);
      const int lbase = kSel2Bins - 32 * (ls + 1);
      // lane j < 32 takes bin lbase + 31 - j (descending)
      const int cj = lane < 32 ? (int)hist[lbase + 31 - lane] : 0;
      const int cinc = wave_inclusive_scan(cj);
      const uint64_t hit2 = __ballot(lane < 32 && ex + cinc >= rank);
      const int js = __builtin_amdgcn_readfirstlane(__ffsll((long long)hit2) - 1);
      if (lane == js) {
        S.res[0] = lbase + 31 - js;
        S.res[1] = ex + cinc - cj;
        S.res[2] = cj;
      }
    } else {
      // clear the other histogram for the next pass while wave 0 scans this one
      uint4* other = reinterpret_cast<uint4*>(S.hist[buf ^ 1]);
      for (int b = t - kWave; b < kSel2Bins / 4; b += NT - kWave) other[b] = make_uint4(0, 0, 0, 0);
    }
    __syncthreads();
    const int bstar = S.res[0], above = S.res[1], cbin = S.res[2];
    rank -= above;
    inrange = cbin;
    const uint32_t nlo = lo + ((uint32_t)bstar << shift);
    hi = (uint32_t)min((uint64_t)hi, (uint64_t)nlo + ((1ull << shift) - 1ull));
    lo = nlo;
    if (shift == 0) {
      r.T = lo;
      r.need_eq = rank;
      r.eq_total = cbin;
      break;
    }
    if (cbin <= kSel2Small) {
      // rank the few keys of this bin directly (one slot reservation per thread)
      int mine_n = 0;
#pragma unroll
      for (int j = 0; j < J; ++j) mine_n += (((cand >> j) & 1ull) && key[j] >= lo && key[j] <= hi) ? 1 : 0;
      if (mine_n) {
        int slot = atomicAdd(&S.nsmall, mine_n);
#pragma unroll
        for (int j = 0; j < J; ++j) {
          if (((cand >> j) & 1ull) && key[j] >= lo && key[j] <= hi) S.small[slot++] = key[j];
        }
      }
      __syncthreads();
      if (w == 0) {
        const uint32_t mine = S.small[lane < cbin ? lane : 0];
        int gt = 0, ge = 0;
        for (int x = 0; x < cbin; ++x) {
          const uint32_t kx = (uint32_t)__builtin_amdgcn_readlane((int)mine, x);
          gt += kx > mine ? 1 : 0;
          ge += kx >= mine ? 1 : 0;
        }
        const uint64_t hit = __ballot(lane < cbin && gt < rank && rank <= ge);
        const int ls = __builtin_amdgcn_readfirstlane(__ffsll((long long)hit) - 1);
        if (lane == ls) {
          S.res[3] = (int)mine;
          S.res[4] = rank - gt;
          S.res[5] = ge - gt;
        }
      }
      __syncthreads();
      r.T = (uint32_t)S.res[3];
      r.need_eq = S.res[4];
      r.eq_total = S.res[5];
      break;
    }
    buf ^= 1;
  }
  return r;
}

// Membership of the slots in the selection, given the threshold: every candidate key
// above T, the first need_eq candidate keys equal to T in slot order, and the `force`
// slots.  Slot (w, j, lane) holds page page[j]; slot order must be ascending page
// order.  *eq_cut receives the page of the last key equal to T that is taken when a tie
// is cut (it is left unchanged otherwise).  Returns this thread's membership mask.
template <int NT, int J>
__device__ __forceinline__ uint64_t sel2_membership(const uint32_t (&key)[J], const int (&page)[J], uint64_t cand,
                                                    uint64_t force, const SelThreshold& th, int* eq_cut, Sel2Lds& S) {
  constexpr int NW = NT / kWave;
  const int lane = lane_id(), w = threadIdx.x / kWave;
  uint64_t gt = 0, eq = 0;
#pragma unroll
  for (int j = 0; j < J; ++j) {
    if ((cand >> j) & 1ull) {
      if (th.mode == 1 || (th.mode == 2 && key[j] > th.T)) gt |= 1ull << j;
      if (th.mode == 2 && key[j] == th.T) eq |= 1ull << j;
    }
  }
  gt |= force;
  if (th.mode != 2 || th.need_eq >= th.eq_total) return gt | eq;  // no tie is cut
  // the first need_eq keys equal to T in slot order
  const int eqc = wave_isum(__popcll(eq));
  __syncthreads();  // S.red may still be read by a previous step
  if (lane == 0) S.red[1][w] = eqc;
  __syncthreads();
  int eq_run = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) eq_run += i < w ? S.red[1][i] : 0;
  uint64_t in = gt;
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const bool e = (eq >> j) & 1ull;
    const uint64_t em = __ballot(e);
    const int erank = eq_run + lanes_below(em);
    if (e && erank < th.need_eq) {
      in |= 1ull << j;
      if (erank == th.need_eq - 1) *eq_cut = page[j];
    }
    eq_run += __popcll(em);
  }
  return in;
}

// The pages of the slots in `mask`, in slot order, to out[0, min(total, cap)) (global or
// LDS); returns the total to every thread.  `wbase`, if not NULL, receives per thread
// the number of masked slots of the waves before this one.
template <int NT, int J>
__device__ __forceinline__ int sel2_list(uint64_t mask, const int (&page)[J], int32_t* __restrict__ out, int cap,
                                         Sel2Lds& S) {
  constexpr int NW = NT / kWave;
  const int lane = lane_id(), w = threadIdx.x / kWave;
  const int c = wave_isum(__popcll(mask));
  __syncthreads();  // S.red may still be read by a previous step
  if (lane == 0) S.red[0][w] = c;
  __syncthreads();
  int run = 0, total = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    const int ci = S.red[0][i];
    run += i < w ? ci : 0;
    total += ci;
  }
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const bool in = (mask >> j) & 1ull;
    const uint64_t bm = __ballot(in);
    if (in) {
      const int pos = run + lanes_below(bm);
      if (pos < cap) out[pos] = page[j];
    }
    run += __popcll(bm);
  }
  return total;
}

// Membership and the list of the selection (ascending pages); the count to *out_count.
template <int NT, int J>
__device__ __forceinline__ uint64_t sel2_compact(const uint32_t (&key)[J], const int (&page)[J], uint64_t cand,
                                                 uint64_t force, const SelThreshold& th, int32_t* __restrict__ out,
                                                 int cap, int32_t* __restrict__ out_count, int* eq_cut, Sel2Lds& S) {
  const uint64_t in = sel2_membership<NT, J>(key, page, cand, force, th, eq_cut, S);
  const int total = sel2_list<NT, J>(in, page, out, cap, S);
  if (threadIdx.x == 0 && out_count) *out_count = min(total, cap);
  return in;
}

}  // namespace prr

namespace prr {

// ------------------------------------------------------------------ one-wave select
// The same exact top-K for at most 64 * NK keys held by ONE wave (slot (j, lane) holds
// page page[j]; slot order j * 64 + lane must be ascending page order).  Used when the
// candidate list is short: a single wave needs no barrier between the radix passes, so
// the threshold is known after a few LDS round trips.  Each wave using it needs its own
// WSelLds.

struct WSelLds {
  uint32_t hist[kSel2Bins];
  uint32_t small[kSel2Small];
};

// The 2048 bins of S, cleared by one wave with contiguous stores.
__device__ __forceinline__ void wsel_clear(WSelLds& S) {
  uint4* hb = reinterpret_cast<uint4*>(S.hist);
#pragma unroll
  for (int v = 0; v < kSel2Bins / 4 / kWave; ++v) hb[v * kWave + lane_id()] = make_uint4(0, 0, 0, 0);
}

// precleared: the bins of S are zero on entry (cleared while the caller waited for the
// keys), so the first pass starts with the atomics.
template <int NK>
__device__ __forceinline__ SelThreshold wsel_threshold(const uint32_t (&key)[NK], uint64_t cand, int kextra,
                                                       WSelLds& S, bool precleared = false) {
  const int lane = lane_id();
  int cnt = __popcll(cand);
  uint32_t lo = 0xffffffffu, hi = 0u;
#pragma unroll
  for (int j = 0; j < NK; ++j) {
    if ((cand >> j) & 1ull) {
      lo = min(lo, key[j]);
      hi = max(hi, key[j]);
    }
  }
  cnt = wave_isum(cnt);
  lo = wave_umin(lo);
  hi = wave_umax(hi);
  SelThreshold r;
  r.mode = 0;
  r.T = 0;
  r.need_eq = 0;
  r.eq_total = 0;
  if (kextra <= 0 || cnt == 0) return r;
  if (kextra >= cnt) {
    r.mode = 1;
    return r;
  }
  r.mode = 2;
  int rank = kextra, inrange = cnt;
  for (int pass = 0; pass < 3; ++pass) {
    const uint32_t range = hi - lo;
    if (range == 0) {
      r.T = lo;
      r.need_eq = rank;
      r.eq_total = inrange;
      return r;
    }
    const int bits = 32 - __clz(range);
    const int shift = bits > kSel2Log2Bins ? bits - kSel2Log2Bins : 0;
    if (pass > 0 || !precleared) {
      wsel_clear(S);
      __builtin_amdgcn_wave_barrier();
    }
    // lane l sums its 32 bins [2048 - 32(l+1), 2048 - 32 l) after the counting
    const int base = kSel2Bins - 32 * (lane + 1);
    const uint4* hb = reinterpret_cast<const uint4*>(S.hist + base);
#pragma unroll
    for (int j = 0; j < NK; ++j)
      if (((cand >> j) & 1ull) && key[j] >= lo && key[j] <= hi) atomicAdd(&S.hist[(key[j] - lo) >> shift], 1u);
    __builtin_amdgcn_wave_barrier();
    int s = 0;
#pragma unroll
    for (int v = 0; v < 8; ++v) {
      const uint4 x = hb[v];
      s += (int)(x.x + x.y + x.z + x.w);
    }
    const int incl = wave_inclusive_scan(s);
    const uint64_t hit = __ballot(incl - s < rank && rank <= incl);
    const int ls = __builtin_amdgcn_readfirstlane(__ffsll((long long)hit) - 1);
    const int ex = __builtin_amdgcn_readlane(incl - s, ls);
    const int lbase = kSel2Bins - 32 * (ls + 1);
    const int cj = lane < 32 ? (int)S.hist[lbase + 31 - lane] : 0;  // descending bins
    const int cinc = wave_inclusive_scan(cj);
    const uint64_t hit2 = __ballot(lane < 32 && ex + cinc >= rank);
    const int js = __builtin_amdgcn_readfirstlane(__ffsll((long long)hit2) - 1);
    const int bstar = lbase + 31 - js;
    const int cbin = __builtin_amdgcn_readlane(cj, js);
    rank -= __builtin_amdgcn_readlane(ex + cinc - cj, js);
    inrange = cbin;
    const uint32_t nlo = lo + ((uint32_t)bstar << shift);
    hi = (uint32_t)min((uint64_t)hi, (uint64_t)nlo + ((1ull << shift) - 1ull));
    lo = nlo;
    if (shift == 0) {
      r.T = lo;
      r.need_eq = rank;
      r.eq_total = cbin;
      return r;
    }
    if (cbin <= 4) {
      // the rank-th largest key of the bin by repeated maxima (cheaper than a compaction
      // for the usual bin of one or two keys); each round takes every key equal to the
      // maximum, so at most cbin rounds
      uint32_t ub = hi;
      for (int round = 0; round < cbin; ++round) {
        uint32_t m = 0u;
#pragma unroll
        for (int j = 0; j < NK; ++j) {
          const bool in = ((cand >> j) & 1ull) && key[j] >= lo && key[j] <= ub;
          m = in ? max(m, key[j] - lo + 1u) : m;
        }
        m = wave_umax(m);  // 1 + (maximum - lo); nonzero while keys remain below ub
        const uint32_t km = lo + m - 1u;
        int c = 0;
#pragma unroll
        for (int j = 0; j < NK; ++j) c += (((cand >> j) & 1ull) && key[j] == km) ? 1 : 0;
        c = wave_isum(c);
        if (rank <= c || m == 0u || km == lo) {
          r.T = km;
          r.need_eq = rank;
          r.eq_total = c;
          return r;
        }
        rank -= c;
        ub = km - 1u;
      }
    }
    if (cbin <= kSel2Small) {
      // the keys of this bin, compacted in slot order, ranked by broadcast
      int pos = 0;
#pragma unroll
      for (int j = 0; j < NK; ++j) {
        const bool in = ((cand >> j) & 1ull) && key[j] >= lo && key[j] <= hi;
        const uint64_t m = __ballot(in);
        if (in) S.small[pos + lanes_below(m)] = key[j];
        pos += __popcll(m);
      }
      __builtin_amdgcn_wave_barrier();
      const uint32_t mine = S.small[lane < cbin ? lane : 0];
      int gt = 0, ge = 0;
      for (int x = 0; x < cbin; ++x) {
        const uint32_t kx = (uint32_t)__builtin_amdgcn_readlane((int)mine, x);
        gt += kx > mine ? 1 : 0;
        ge += kx >= mine ? 1 : 0;
      }
      const uint64_t hit3 = __ballot(lane < cbin && gt < rank && rank <= ge);
      const int l3 = __builtin_amdgcn_readfirstlane(__ffsll((long long)hit3) - 1);
      r.T = (uint32_t)__builtin_amdgcn_readlane((int)mine, l3);
      r.need_eq = rank - __builtin_amdgcn_readlane(gt, l3);
      r.eq_total = __builtin_amdgcn_readlane(ge - gt, l3);
      return r;
    }
    __builtin_amdgcn_wave_barrier();
  }
  r.T = lo;
  r.need_eq = rank;
  r.eq_total = inrange;
  return r;
}

// Membership given the threshold (one wave; ties cut in slot order).  *eq_cut (written by
// one lane) receives the page of the last key equal to T that is taken when a tie is cut.
template <int NK>
__device__ __forceinline__ uint64_t wsel_membership(const uint32_t (&key)[NK], const int (&page)[NK], uint64_t cand,
                                                    uint64_t force, const SelThreshold& th, int* eq_cut) {
  uint64_t gt = 0, eq = 0;
#pragma unroll
  for (int j = 0; j < NK; ++j) {
    if ((cand >> j) & 1ull) {
      if (th.mode == 1 || (th.mode == 2 && key[j] > th.T)) gt |= 1ull << j;
      if (th.mode == 2 && key[j] == th.T) eq |= 1ull << j;
    }
  }
  gt |= force;
  if (th.mode != 2 || th.need_eq >= th.eq_total) return gt | eq;
  uint64_t in = gt;
  int run = 0;
#pragma unroll
  for (int j = 0; j < NK; ++j) {
    const bool e = (eq >> j) & 1ull;
    const uint64_t em = __ballot(e);
    const int er = run + lanes_below(em);
    if (e && er < th.need_eq) {
      in |= 1ull << j;
      if (er == th.need_eq - 1) *eq_cut = page[j];
    }
    run += __popcll(em);
  }
  return in;
}

}  // namespace prr

namespace prr {

// ------------------------------------------------------------ block select of <= 1024 keys
// The threshold of the same exact top-K for at most 2 * NT keys, two per thread, without
// gathering them into one wave: every pass builds the histogram of the current key range
// with LDS atomics, scans it (four bins per thread, DPP prefix within the wave, wave
// totals through LDS) and keeps the bin holding the wanted rank, until that bin holds a
// single key or a single value.  The bins of `hist` must be zero on entry (they are left
// nonzero).

struct BSelLds {
  uint32_t hist[kSel2Bins];
  uint32_t red[2][16];
  int res[4];
};

template <int NT>
__device__ __forceinline__ SelThreshold bsel_threshold(const uint32_t (&key)[2], const bool (&cand)[2], int kextra,
                                                       BSelLds& S) {
  static_assert(NT == 512, "four bins per thread");
  constexpr int NW = NT / kWave;
  const int t = threadIdx.x, lane = lane_id(), w = t / kWave;
  uint32_t lo = 0xffffffffu, hi = 0u;
  int cnt = 0;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    if (cand[j]) {
      lo = min(lo, key[j]);
      hi = max(hi, key[j]);
      ++cnt;
    }
  }
  lo = wave_umin(lo);
  hi = wave_umax(hi);
  cnt = wave_isum(cnt);
  if (lane == 0) {
    S.red[0][w] = lo;
    S.red[1][w] = hi;
    S.red[0][NW + w] = (uint32_t)cnt;
  }
  __syncthreads();
  cnt = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    lo = min(lo, S.red[0][i]);
    hi = max(hi, S.red[1][i]);
    cnt += (int)S.red[0][NW + i];
  }
  SelThreshold r;
  r.mode = 0;
  r.T = 0;
  r.need_eq = 0;
  r.eq_total = 0;
  if (kextra <= 0 || cnt == 0) return r;
  if (kextra >= cnt) {
    r.mode = 1;
    return r;
  }
  r.mode = 2;
  int rank = kextra, inrange = cnt;
  // thread t owns bins [2048 - 4(t+1), 2048 - 4t) (bins in descending key order)
  const int b0 = kSel2Bins - 4 * (t + 1);
  for (int pass = 0; pass < 3; ++pass) {
    const uint32_t range = hi - lo;
    if (range == 0) break;
    const int bits = 32 - __clz(range);
    const int shift = bits > kSel2Log2Bins ? bits - kSel2Log2Bins : 0;
    if (pass > 0) {
      reinterpret_cast<uint4*>(S.hist)[t] = make_uint4(0, 0, 0, 0);
      __syncthreads();
    }
#pragma unroll
    for (int j = 0; j < 2; ++j)
      if (cand[j] && key[j] >= lo && key[j] <= hi) atomicAdd(&S.hist[(key[j] - lo) >> shift], 1u);
    __syncthreads();
    const uint4 hv = reinterpret_cast<const uint4*>(S.hist)[b0 / 4];
    const int s = (int)(hv.x + hv.y + hv.z + hv.w);
    const int incl = wave_inclusive_scan(s);
    if (lane == kWave - 1) S.red[1][w] = (uint32_t)incl;
    __syncthreads();
    int before = incl - s;
#pragma unroll
    for (int i = 0; i < NW; ++i) before += i < w ? (int)S.red[1][i] : 0;
    if (before < rank && rank <= before + s) {
      // descending: bins b0+3, b0+2, b0+1, b0
      const int c3 = (int)hv.w, c2 = (int)hv.z, c1 = (int)hv.y;
      int bstar, above;
      if (rank <= before + c3) {
        bstar = b0 + 3;
        above = before;
      } else if (rank <= before + c3 + c2) {
        bstar = b0 + 2;
        above = before + c3;
      } else if (rank <= before + c3 + c2 + c1) {
        bstar = b0 + 1;
        above = before + c3 + c2;
      } else {
        bstar = b0;
        above = before + c3 + c2 + c1;
      }
      S.res[0] = bstar;
      S.res[1] = above;
      S.res[2] = (int)S.hist[bstar];
      S.res[3] = 0;  // the compaction counter of a small bin
    }
    __syncthreads();
    const int bstar = S.res[0], cbin = S.res[2];
    rank -= S.res[1];
    inrange = cbin;
    const uint32_t nlo = lo + ((uint32_t)bstar << shift);
    hi = (uint32_t)min((uint64_t)hi, (uint64_t)nlo + ((1ull << shift) - 1ull));
    lo = nlo;
    if (shift == 0) break;
    if (cbin == 1) {
      // the single key of the bin is T: its holder publishes it
#pragma unroll
      for (int j = 0; j < 2; ++j)
        if (cand[j] && key[j] >= lo && key[j] <= hi) S.res[3] = (int)key[j];
      __syncthreads();
      r.T = (uint32_t)S.res[3];
      r.need_eq = rank;
      r.eq_total = 1;
      return r;
    }
    if (cbin <= kWave) {
      // Few keys in the bin that holds rank K: they go to LDS (the histogram is read no
      // more) and one wave ranks them, instead of another histogram pass.  T is the
      // rank-th largest of them; the keys equal to T all lie in this bin.
#pragma unroll
      for (int j = 0; j < 2; ++j)
        if (cand[j] && key[j] >= lo && key[j] <= hi) S.hist[atomicAdd(&S.res[3], 1)] = key[j];
      __syncthreads();
      if (w == 0) {
        const int nb = min(S.res[3], kWave);
        const uint32_t mk = lane < nb ? S.hist[lane] : 0u;
        int gt = 0, eq = 0;
        for (int j = 0; j < nb; ++j) {  // (the keys from registers: no LDS round trip per key)
          const uint32_t o = (uint32_t)__builtin_amdgcn_readlane((int)mk, j);
          gt += o > mk ? 1 : 0;
          eq += o == mk ? 1 : 0;
        }
        if (lane < nb && gt < rank && rank <= gt + eq) {  // (every lane holding T writes the same)
          S.red[0][0] = mk;
          S.red[0][1] = (uint32_t)(rank - gt);
          S.red[0][2] = (uint32_t)eq;
        }
      }
      __syncthreads();
      r.T = S.red[0][0];
      r.need_eq = (int)S.red[0][1];
      r.eq_total = (int)S.red[0][2];
      return r;
    }
  }
  // a bin of one value (or three passes): every key in [lo, hi] equals lo
  r.T = lo;
  r.need_eq = rank;
  r.eq_total = inrange;
  return r;
}

}  // namespace prr
