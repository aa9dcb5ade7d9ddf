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
      // lane l owns bins [2048 - 32(l+1), 2048 - 32l); c[i] is bin base + i
      const int base = kSel2Bins - 32 * (lane + 1);
      uint32_t c[32];
      const uint4* hb = reinterpret_cast<const uint4*>(hist + base);
#pragma unroll
      for (int v = 0; v < 8; ++v) {
        const uint4 x = hb[v];
        c[4 * v] = x.x;
        c[4 * v + 1] = x.y;
        c[4 * v + 2] = x.z;
        c[4 * v + 3] = x.w;
      }
      int s = 0;
#pragma unroll
      for (int i = 0; i < 32; ++i) s += (int)c[i];
      const int incl = wave_inclusive_scan(s);
      const int excl = incl - s;
      if (excl < rank && rank <= incl) {
        int run = excl;
        bool found = false;
#pragma unroll
        for (int i = 31; i >= 0; --i) {
          const int ci = (int)c[i];
          if (!found && run + ci >= rank) {
            S.res[0] = base + i;
            S.res[1] = run;
            S.res[2] = ci;
            found = true;
          }
          run += ci;
        }
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
      // rank the few keys of this bin directly
#pragma unroll
      for (int j = 0; j < J; ++j) {
        if (((cand >> j) & 1ull) && key[j] >= lo && key[j] <= hi) S.small[atomicAdd(&S.nsmall, 1)] = key[j];
      }
      __syncthreads();
      if (w == 0) {
        const uint32_t mine = S.small[lane < cbin ? lane : 0];
        int gt = 0, ge = 0;
        const uint4* sv = reinterpret_cast<const uint4*>(S.small);
#pragma unroll
        for (int v = 0; v < kSel2Small / 4; ++v) {
          const uint4 x = sv[v];
          const uint32_t xs[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const bool live = 4 * v + e < cbin;
            gt += (live && xs[e] > mine) ? 1 : 0;
            ge += (live && xs[e] >= mine) ? 1 : 0;
          }
        }
        if (lane < cbin && gt < rank && rank <= ge) {
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

// Membership of the candidates in the selection, given the threshold: every key above
// T, and keys equal to T up to need_eq of them in page order.  `force` pages are added.
// Writes the selected pages in ascending order to out[0, min(total, cap)), the count
// to *out_count (thread 0), and returns this thread's membership mask.  *eq_cut
// receives the page of the last key equal to T that is taken (or is left unchanged
// when no tie is cut).
template <int NT, int J>
__device__ __forceinline__ uint64_t sel2_compact(const uint32_t (&key)[J], uint64_t cand, uint64_t force, const SelThreshold& th,
                                 int32_t* __restrict__ out, int cap, int32_t* __restrict__ out_count, int* eq_cut,
                                 Sel2Lds& S) {
  constexpr int NW = NT / kWave;
  const int t = threadIdx.x, lane = lane_id(), w = t / kWave;
  uint64_t gt = 0, eq = 0;
#pragma unroll
  for (int j = 0; j < J; ++j) {
    if ((cand >> j) & 1ull) {
      if (th.mode == 1 || (th.mode == 2 && key[j] > th.T)) gt |= 1ull << j;
      if (th.mode == 2 && key[j] == th.T) eq |= 1ull << j;
    }
  }
  gt |= force;
  const int gtc = wave_isum(__popcll(gt)), eqc = wave_isum(__popcll(eq));
  __syncthreads();  // S.red may still be read by a previous step
  if (lane == 0) {
    S.red[0][w] = gtc;
    S.red[1][w] = eqc;
  }
  __syncthreads();
  int eq_run = 0, sel_run = 0, total = 0;
  {
    int eb = 0, sb = 0;
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      const int gi = S.red[0][i], ei = S.red[1][i];
      const int take = max(0, min(ei, th.need_eq - eb));
      if (i == w) {
        eq_run = eb;
        sel_run = sb;
      }
      eb += ei;
      sb += gi + take;
    }
    total = sb;
  }
  uint64_t in = 0;
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const bool e = (eq >> j) & 1ull;
    const uint64_t em = __ballot(e);
    const int erank = eq_run + lanes_below(em);
    const bool take_eq = e && erank < th.need_eq;
    const bool sel = ((gt >> j) & 1ull) || take_eq;
    const uint64_t sm = __ballot(sel);
    if (sel) {
      const int pos = sel_run + lanes_below(sm);
      if (out && pos < cap) out[pos] = sel2_page<J>(j);
      in |= 1ull << j;
    }
    if (take_eq && erank == th.need_eq - 1 && th.need_eq < th.eq_total) *eq_cut = sel2_page<J>(j);
    eq_run += __popcll(em);
    sel_run += __popcll(sm);
  }
  if (t == 0 && out_count) *out_count = min(total, cap);
  return in;
}

}  // namespace prr
