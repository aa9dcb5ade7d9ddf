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
#include "prr_device.h"
#include "prr_launch.h"
#include "prr_select.h"

namespace prr {

typedef __attribute__((ext_vector_type(4))) uint32_t u32x4_t;

namespace {

constexpr int kFT = 512;
constexpr int kFW = kFT / kWave;
constexpr int kFScorePages = 128;
constexpr int kFSpin = 1 << 20;
constexpr int kFPart = kHeadDim + 2;  // o[128], m, l of one query head
constexpr uint32_t kSelfMiss = 0x80000000u;
constexpr int kFOPad = kHeadDim + 4;
constexpr int kEqAll = 16383;  // eq_cut meaning "every key equal to T is taken"

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
    __builtin_amdgcn_s_sleep(1);
    v = get_tag(p);
  }
  if (!tag_is(v, epoch)) atomicOr(flags, kFlagSpinTimeout);
  return (uint32_t)v;
}
__device__ __forceinline__ uint32_t wait_tag(const uint64_t* p, uint32_t epoch, uint32_t* flags) {
  return tagged(get_tag(p), p, epoch, flags);
}

// ------------------------------------------------------------------------ LDS

struct FScoreLds {
  float qpart[16][kHeadDim];
  float qbar[kHeadDim];
};

struct FSelLds {
  Sel2Lds sel;
  uint32_t bitP[PRR_MAX_PAGES_DEV / 32];
  uint32_t forceb[PRR_MAX_PAGES_DEV / 32];
  int32_t mlist[PRR_MAX_CAP_DEV];
  int cnt[2][16];
  int eq_cut;
};

struct FAttnLds {
  float wo[kFW][16][kFOPad];
  float wm[kFW][16];
  float wl[kFW][16];
};

struct FMergeLds {
  float w[2 * PRR_MAX_CAP_DEV];  // l, then the weight, of each state
  float m[2 * PRR_MAX_CAP_DEV];
  float red[2][kFW];
  float acc[4][kHeadDim];
};

union FLds {
  FScoreLds score;
  FSelLds sel;
  FAttnLds attn;
  FMergeLds merge;
};

// ------------------------------------------------------------------------ score

template <bool BF16>
__device__ __forceinline__ void role_score(const FusedLaunch& a, int h, int blk, FScoreLds& S) {
  const int t = threadIdx.x, lane = lane_id(), w = t / kWave;
  const int G = a.group;
  const uint16_t* q = static_cast<const uint16_t*>(a.q);
  {
    const int g = t >> 4, c8 = (t & 15) * 8;
    if (g < G) {
      const uint4 v = *reinterpret_cast<const uint4*>(q + (size_t)(h * G + g) * kHeadDim + c8);
#pragma unroll
      for (int e = 0; e < 8; ++e) S.qpart[g][c8 + e] = u4_elem<BF16>(v, e);
    }
    __syncthreads();
    if (t < kHeadDim) {
      float s = 0.0f;
      for (int gg = 0; gg < G; ++gg) s += S.qpart[gg][t];
      S.qbar[t] = s / (float)G;
    }
    __syncthreads();
  }
  const int cg = lane & 15, pi = lane >> 4;
  float qb[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) qb[e] = S.qbar[cg * 8 + e];
  const int base = blk * kFScorePages + w * 16 + pi;
  const int n = a.num_pages;
  float* scores = a.scores + (size_t)h * a.max_pages;
  uint64_t* ts = a.t_score + (size_t)h * a.max_pages;
  float s[4];
  if (!a.meta_mean) {
    uint4 mn[4], mx[4];
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      const int p = min(base + 4 * it, n - 1);
      const uint16_t* row = static_cast<const uint16_t*>(a.meta) + ((size_t)h * a.max_pages + p) * 2 * kHeadDim + cg * 8;
      mn[it] = *reinterpret_cast<const uint4*>(row);
      mx[it] = *reinterpret_cast<const uint4*>(row + kHeadDim);
    }
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      float v = 0.0f;
#pragma unroll
      for (int e = 0; e < 8; ++e) v += fmaxf(qb[e] * u4_elem<BF16>(mn[it], e), qb[e] * u4_elem<BF16>(mx[it], e));
      s[it] = v;
    }
  } else {
    float4 m0[4], m1[4];
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      const int p = min(base + 4 * it, n - 1);
      const float4* row = reinterpret_cast<const float4*>(static_cast<const float*>(a.meta) +
                                                          ((size_t)h * a.max_pages + p) * kHeadDim + cg * 8);
      m0[it] = row[0];
      m1[it] = row[1];
    }
#pragma unroll
    for (int it = 0; it < 4; ++it) {
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
  for (int it = 0; it < 4; ++it) {
    const float v = sum16(s[it]);
    const int p = base + 4 * it;
    if (cg == 0 && p < n) {
      scores[p] = v;
      put_tag(&ts[p], __float_as_uint(v), a.epoch);
    }
  }
}

// ------------------------------------------------------------------------ shared select pieces

// This thread's J scores of KV head h, polled until every one carries this epoch.
template <int J>
__device__ __forceinline__ void poll_scores(const FusedLaunch& a, int h, uint32_t (&sb)[J]) {
  const int n = a.num_pages;
  const uint64_t* ts = a.t_score + (size_t)h * a.max_pages;
  uint64_t pending = 0;
#pragma unroll
  for (int j = 0; j < J; ++j) {
    sb[j] = 0u;
    if (sel2_page<J>(j) < n) pending |= 1ull << j;
  }
  for (int it = 0; pending && it < kFSpin; ++it) {
    uint64_t v[J];
#pragma unroll
    for (int j = 0; j < J; ++j) v[j] = get_tag(&ts[min(sel2_page<J>(j), n - 1)]);
#pragma unroll
    for (int j = 0; j < J; ++j) {
      if (((pending >> j) & 1ull) && tag_is(v[j], a.epoch)) {
        sb[j] = (uint32_t)v[j];
        pending &= ~(1ull << j);
      }
    }
    if (pending) __builtin_amdgcn_s_sleep(1);
  }
  if (pending) atomicOr(a.flags, kFlagSpinTimeout);
}

__device__ __forceinline__ void forced_bitmap(const FusedLaunch& a, uint32_t* forceb) {
  const int t = threadIdx.x;
  const int nw = (a.num_pages + 31) >> 5;
  for (int i = t; i < nw; i += kFT) forceb[i] = 0u;
  __syncthreads();
  // the forced list lives in the kernel arguments: read it with constant indices only
  if (t == 0) {
#pragma unroll
    for (int i = 0; i < PRR_MAX_FORCED; ++i)
      if (i < a.n_forced) atomicOr(&forceb[a.forced[i] >> 5], 1u << (a.forced[i] & 31));
  }
  __syncthreads();
}

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

template <bool BF16>
__device__ __forceinline__ float v_elem(const u32x4_t& v, int e) {
  const uint32_t w = v[e >> 1];
  return h2f<BF16>((e & 1) ? (w >> 16) : (w & 0xffffu));
}

// q.k^T of a 16-token tile as four 16x16x32 MFMAs with the contraction index permuted so
// that lane 16j+r reads 64 contiguous bytes of its key row (channels 32j..32j+31); the
// result gives lane 16j+n the logits of tokens 4j..4j+3 for head n.  p.V is computed
// transposed, O^T += V^T P^T, as 32 fp32 16x16x4 MFMAs (weights stay fp32): call
// (tg, cb) contracts tokens {tg, 4+tg, 8+tg, 12+tg}, lane 16j+m supplying
// V[4j+tg][8m+cb] and p[head n][4j+tg].
template <bool BF16, int PS, int NPW>
__device__ __forceinline__ void wave_attend(const FusedLaunch& a, int h, const int (&pg)[NPW], WaveStates<NPW>& st) {
  constexpr int TPP = PS / 16;
  constexpr int NTW = NPW * TPP;
  const float kNegInf = -__builtin_inff();
  const float scale = 0.08838834764831845f;  // 1/sqrt(128)
  const int lane = lane_id(), j = lane >> 4, n = lane & 15;
  const int G = a.group;
  const uint16_t* qh = static_cast<const uint16_t*>(a.q) + (size_t)h * G * kHeadDim;
  const uint16_t* kh = static_cast<const uint16_t*>(a.k_cache) + (size_t)h * a.max_pages * PS * kHeadDim;
  const uint16_t* vh = static_cast<const uint16_t*>(a.v_cache) + (size_t)h * a.max_pages * PS * kHeadDim;

  u32x4_t qf[4];
  if (n < G) {
    const u32x4_t* src = reinterpret_cast<const u32x4_t*>(qh + (size_t)n * kHeadDim + 32 * j);
#pragma unroll
    for (int s = 0; s < 4; ++s) qf[s] = src[s];
  } else {
#pragma unroll
    for (int s = 0; s < 4; ++s) qf[s] = u32x4_t{0, 0, 0, 0};
  }
  int phys[NPW];
#pragma unroll
  for (int k = 0; k < NPW; ++k) phys[k] = (pg[k] >= 0 && a.page_table) ? a.page_table[pg[k]] : pg[k];
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
    if (tt > 0) {
#pragma unroll
      for (int cb = 0; cb < 8; ++cb) {
#pragma unroll
        for (int i = 0; i < 4; ++i) st.acc[k][cb][i] *= alpha;
      }
    }
#pragma unroll
    for (int tg = 0; tg < 4; ++tg) {
#pragma unroll
      for (int cb = 0; cb < 8; ++cb)
        st.acc[k][cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(v_elem<BF16>(vf[f][tg], cb), p[tg], st.acc[k][cb], 0, 0, 0);
    }
  }
}

// Fold the kept page states of every wave (keep: wave-uniform bit mask) and publish the
// workgroup's state into partial slot `slot` of KV head h.
template <int NPW>
__device__ __forceinline__ void fold_publish(const FusedLaunch& a, int h, int slot, WaveStates<NPW>& st, uint32_t keep,
                             FAttnLds& L) {
  const float kNegInf = -__builtin_inff();
  const int t = threadIdx.x, lane = lane_id(), w = t / kWave;
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
  __syncthreads();
  const int hh = t >> 5, c0 = (t & 31) * 4;
  const int G = a.group;
  if (hh < G) {
    float mw[kFW], fw[kFW];
    float ms = kNegInf;
#pragma unroll
    for (int ww = 0; ww < kFW; ++ww) {
      mw[ww] = L.wm[ww][hh];
      if (L.wl[ww][hh] > 0.0f) ms = fmaxf(ms, mw[ww]);
    }
    float lsum = 0.0f;
#pragma unroll
    for (int ww = 0; ww < kFW; ++ww) {
      const float lw = L.wl[ww][hh];
      fw[ww] = lw > 0.0f ? exp2f((mw[ww] - ms) * kLog2e) : 0.0f;
      lsum += lw * fw[ww];
    }
    const float inv = lsum > 0.0f ? 1.0f / lsum : 0.0f;
    float o[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ww = 0; ww < kFW; ++ww) {
      const float4 x = *reinterpret_cast<const float4*>(&L.wo[ww][hh][c0]);
      o[0] += x.x * fw[ww];
      o[1] += x.y * fw[ww];
      o[2] += x.z * fw[ww];
      o[3] += x.w * fw[ww];
    }
    uint64_t* dst = a.t_part + (((size_t)h * a.nparts + slot) * G + hh) * kFPart;
#pragma unroll
    for (int e = 0; e < 4; ++e) put_tag(dst + c0 + e, __float_as_uint(o[e] * inv), a.epoch);
    if ((t & 31) == 0) {
      put_tag(dst + kHeadDim, __float_as_uint(lsum > 0.0f ? ms : kNegInf), a.epoch);
      put_tag(dst + kHeadDim + 1, __float_as_uint(lsum), a.epoch);
    }
  }
}

__device__ __forceinline__ bool page_forced(const FusedLaunch& a, int p) {
  bool f = false;
#pragma unroll
  for (int i = 0; i < PRR_MAX_FORCED; ++i) f |= i < a.n_forced && a.forced[i] == p;
  return f;
}

// ------------------------------------------------------------------------ select

template <bool BF16, int PS, int J>
__device__ __forceinline__ void role_select(const FusedLaunch& a, int h, FLds& U) {
  FSelLds& L = U.sel;
  const int t = threadIdx.x, lane = lane_id(), w = t / kWave;
  const int n = a.num_pages, nw = (n + 31) >> 5;
  const bool prr = a.schedule == 1;
  // bitmaps of the forced pages and of P^t
  for (int i = t; i < nw; i += kFT) {
    L.forceb[i] = 0u;
    L.bitP[i] = 0u;
  }
  if (t == 0) L.eq_cut = kEqAll;
  __syncthreads();
  if (t == 0) {
#pragma unroll
    for (int i = 0; i < PRR_MAX_FORCED; ++i)
      if (i < a.n_forced) atomicOr(&L.forceb[a.forced[i] >> 5], 1u << (a.forced[i] & 31));
  }
  if (prr) {
    const int pc = min(max(a.pred_cur_count[h], 0), a.cap);
    for (int i = t; i < pc; i += kFT) {
      const int p = a.pred_cur[(size_t)h * a.cap + i];
      if (p >= 0 && p < n) atomicOr(&L.bitP[p >> 5], 1u << (p & 31));
    }
  }
  __syncthreads();

  uint32_t sb[J];
  poll_scores<J>(a, h, sb);
  uint32_t key[J];
  uint64_t cand = 0, force = 0, inP = 0;
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int p = sel2_page<J>(j);
    const int pc = min(p, n - 1);
    key[j] = score_key(__uint_as_float(sb[j]));
    const bool f = p < n && bit_of(L.forceb, pc);
    if (p < n && !f) cand |= 1ull << j;
    if (f) force |= 1ull << j;
    if (p < n && bit_of(L.bitP, pc)) inP |= 1ull << j;
  }
  const SelThreshold th = sel2_threshold<kFT, J>(key, cand, a.kextra_a, L.sel);
  const bool early = th.mode != 2 || th.need_eq == th.eq_total;
  uint64_t* thr = a.t_thr + 2 * (size_t)h;
  if (prr && early && t == 0) {
    put_tag(thr, th.T, a.epoch);
    put_tag(thr + 1, (uint32_t)th.mode | ((uint32_t)kEqAll << 2), a.epoch);
  }
  const uint64_t inA = sel2_compact<kFT, J>(key, cand, force, th, a.selected + (size_t)h * a.cap, a.cap,
                                            a.selected_count + h, &L.eq_cut, L.sel);
  __syncthreads();
  if (prr && !early && t == 0) {
    put_tag(thr, th.T, a.epoch);
    put_tag(thr + 1, (uint32_t)th.mode | ((uint32_t)L.eq_cut << 2), a.epoch);
  }

  // the list to attend after selection: A \ P (PRR) or A (serial), in page order
  const uint64_t inM = prr ? (inA & ~inP) : inA;
  const uint64_t inW = prr ? (inP & ~inA) : 0ull;
  const int mc = wave_isum(__popcll(inM)), wc = wave_isum(__popcll(inW));
  if (lane == 0) {
    L.cnt[0][w] = mc;
    L.cnt[1][w] = wc;
  }
  __syncthreads();
  int mbase = 0, nM = 0, nW = 0;
#pragma unroll
  for (int i = 0; i < kFW; ++i) {
    mbase += i < w ? L.cnt[0][i] : 0;
    nM += L.cnt[0][i];
    nW += L.cnt[1][i];
  }
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const bool in = (inM >> j) & 1ull;
    const uint64_t bm = __ballot(in);
    if (in) {
      const int pos = mbase + lanes_below(bm);
      if (pos < a.cap) L.mlist[pos] = sel2_page<J>(j);
    }
    mbase += __popcll(bm);
  }
  nM = min(nM, a.cap);
  if (t == 0) {
    if (a.missed_count) a.missed_count[h] = nM;
    if (a.wasted_count) a.wasted_count[h] = nW;
  }
  __syncthreads();
  if (nM == 0) {
    if (t == 0) put_tag(&a.t_mcnt[h], 0u, a.epoch);
  } else if (nM <= kFW) {
    // few enough to attend here: one page per wave, published as the first miss slot
    if (t == 0) put_tag(&a.t_mcnt[h], (uint32_t)nM | kSelfMiss, a.epoch);
    int pg[1];
    pg[0] = __builtin_amdgcn_readfirstlane(w < nM ? L.mlist[w] : -1);
    __syncthreads();  // the list is read before the attention reuses the LDS
    WaveStates<1> st;
    wave_attend<BF16, PS, 1>(a, h, pg, st);
    fold_publish<1>(a, h, a.n_spec, st, 1u, U.attn);
  } else {
    uint64_t* ml = a.t_mlist + (size_t)h * a.cap;
    for (int i = t; i < nM; i += kFT) put_tag(&ml[i], (uint32_t)L.mlist[i], a.epoch);
    if (t == 0) put_tag(&a.t_mcnt[h], (uint32_t)nM, a.epoch);
  }
}

// ------------------------------------------------------------------------ predict

template <int J>
__device__ __forceinline__ void role_predict(const FusedLaunch& a, int h, FLds& U) {
  FSelLds& L = U.sel;
  const int lane = lane_id();
  const int n = a.num_pages;
  forced_bitmap(a, L.forceb);
  uint32_t sb[J];
  poll_scores<J>(a, h, sb);
  const int nwmax = (a.max_pages + 31) / 32;
  float* level = a.level + (size_t)h * a.max_pages;
  float* trend = a.trend + (size_t)h * a.max_pages;
  uint32_t* bits = a.init_bits + (size_t)h * nwmax;
  uint32_t key[J];
  uint64_t cand = 0, force = 0;
  constexpr int JB = J < 16 ? J : 16;  // EMA state is loaded in batches of 16 keys per thread
#pragma unroll
  for (int j0 = 0; j0 < J; j0 += JB) {
    float lv[JB], tv[JB];
    uint32_t bw[JB];
#pragma unroll
    for (int jj = 0; jj < JB; ++jj) {
      const int p = min(sel2_page<J>(j0 + jj), n - 1);
      lv[jj] = level[p];
      tv[jj] = trend[p];
      bw[jj] = bits[p >> 5];
    }
#pragma unroll
    for (int jj = 0; jj < JB; ++jj) {
      const int j = j0 + jj;
      const int p = sel2_page<J>(j);
      const bool inr = p < n;
      bool has = inr && ((bw[jj] >> (p & 31)) & 1u);
      float l = lv[jj], v = tv[jj];
      if (inr) {
        const float s = __uint_as_float(sb[j]);
        if (has) {
          v = a.beta * (s - l) + (1.0f - a.beta) * v;  // Eq. (3): the trend reads the previous level
          l = a.alpha * s + (1.0f - a.alpha) * l;
        } else {
          l = s;
          v = 0.0f;
          has = true;
        }
        level[p] = l;
        trend[p] = v;
      }
      key[j] = score_key(l + a.gamma * v);  // Eq. (2)
      const bool f = inr && bit_of(L.forceb, p);
      if (has && !f) cand |= 1ull << j;
      if (f) force |= 1ull << j;
      const uint64_t hm = __ballot(has);
      const uint64_t vm = __ballot(inr);
      if (lane == 0 || lane == 32) {
        const uint32_t hbits = (uint32_t)(lane == 0 ? hm : (hm >> 32));
        const uint32_t vbits = (uint32_t)(lane == 0 ? vm : (vm >> 32));
        if (vbits) bits[p >> 5] = (bw[jj] & ~vbits) | hbits;
      }
    }
  }
  const SelThreshold th = sel2_threshold<kFT, J>(key, cand, a.kextra_p, L.sel);
  sel2_compact<kFT, J>(key, cand, force, th, a.pred_nxt + (size_t)h * a.cap, a.cap, a.pred_nxt_count + h,
                       &L.eq_cut, L.sel);
}

// ------------------------------------------------------------------------ spec / miss

template <bool BF16, int PS, int NPW>
__device__ __forceinline__ void role_spec(const FusedLaunch& a, int h, int c, FLds& U) {
  const int count = min(max(a.pred_cur_count[h], 0), a.cap);
  const int start = c * a.chunk;
  if (start >= count) return;
  const int cnt = min(a.chunk, count - start);
  const int w = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
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
  wave_attend<BF16, PS, NPW>(a, h, pg, st);
  if (a.mode == PRR_EXACT_SELECTED && keep) {
    // membership of this wave's pages in A, from their scores and the published
    // threshold (all loads issued together, then waited for)
    const uint64_t* ts = a.t_score + (size_t)h * a.max_pages;
    const uint64_t* thr = a.t_thr + 2 * (size_t)h;
    uint64_t vs[NPW];
#pragma unroll
    for (int k = 0; k < NPW; ++k) vs[k] = get_tag(&ts[max(pg[k], 0)]);
    const uint64_t v0 = get_tag(thr), v1 = get_tag(thr + 1);
    uint32_t sc[NPW];
#pragma unroll
    for (int k = 0; k < NPW; ++k) sc[k] = pg[k] >= 0 ? tagged(vs[k], &ts[pg[k]], a.epoch, a.flags) : 0u;
    const uint32_t T = tagged(v0, thr, a.epoch, a.flags);
    const uint32_t me = tagged(v1, thr + 1, a.epoch, a.flags);
    const int mode = (int)(me & 3u), eq_cut = (int)(me >> 2);
#pragma unroll
    for (int k = 0; k < NPW; ++k) {
      if (pg[k] < 0 || page_forced(a, pg[k])) continue;
      const uint32_t key = score_key(__uint_as_float(sc[k]));
      const bool in = mode == 1 || (mode == 2 && (key > T || (key == T && pg[k] <= eq_cut)));
      if (!in) keep &= ~(1u << k);
    }
  }
  fold_publish<NPW>(a, h, c, st, keep, U.attn);
}

template <bool BF16, int PS, int NPW>
__device__ __forceinline__ void role_miss(const FusedLaunch& a, int h, int u, FLds& U) {
  // the count and this wave's list entries are loaded together; the entries are
  // published before the count, so they are usually valid when the count is
  const int start = u * a.chunk;
  const int w = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
  const uint64_t* ml = a.t_mlist + (size_t)h * a.cap;
  uint64_t ve[NPW];
#pragma unroll
  for (int k = 0; k < NPW; ++k) ve[k] = get_tag(&ml[min(start + w + kFW * k, a.cap - 1)]);
  const uint32_t mv = wait_tag(a.t_mcnt + h, a.epoch, a.flags);
  if (mv & kSelfMiss) return;
  const int nM = (int)(mv & ~kSelfMiss);
  if (start >= nM) return;
  const int cnt = min(a.chunk, nM - start);
  int pg[NPW];
  uint32_t keep = 0;
#pragma unroll
  for (int k = 0; k < NPW; ++k) {
    const int i = w + kFW * k;
    int p = i < cnt ? (int)tagged(ve[k], &ml[start + i], a.epoch, a.flags) : -1;
    p = __builtin_amdgcn_readfirstlane(p);
    if (i < cnt && (p < 0 || p >= a.num_pages)) {  // only after a timed-out wait
      if (lane_id() == 0) atomicOr(a.flags, kFlagBadListEntry);
      p = -1;
    }
    pg[k] = p;
    if (p >= 0) keep |= 1u << k;
  }
  WaveStates<NPW> st;
  wave_attend<BF16, PS, NPW>(a, h, pg, st);
  fold_publish<NPW>(a, h, a.n_spec + u, st, keep, U.attn);
}

// ------------------------------------------------------------------------ merge

template <bool BF16>
__device__ __forceinline__ void role_merge(const FusedLaunch& a, int h, int qn, FMergeLds& L) {
  const float kNegInf = -__builtin_inff();
  const int t = threadIdx.x, lane = lane_id(), w = t / kWave;
  const int G = a.group, C = a.chunk;
  int nspec = 0;
  if (a.schedule == 1) nspec = (min(max(a.pred_cur_count[h], 0), a.cap) + C - 1) / C;
  const uint32_t mv = wait_tag(a.t_mcnt + h, a.epoch, a.flags);
  const int nM = (int)(mv & ~kSelfMiss);
  const int nmiss = (mv & kSelfMiss) ? 1 : (nM + C - 1) / C;
  const int total = nspec + nmiss;
  // state i lives in slot i (speculation chunks) or n_spec + (i - nspec) (missed chunks)
  const uint64_t* part = a.t_part + ((size_t)h * a.nparts * G + qn) * kFPart;
  const size_t sstride = (size_t)G * kFPart;
  const int slot_gap = a.n_spec - nspec;
#define PRR_ELEM(i, idx) (part + (size_t)((i) < nspec ? (i) : (i) + slot_gap) * sstride + (idx))

  // This thread's output values of states g, g+4, .. (batches of 16) and the (m, l) of
  // states t, t+512, ..: the first batch and every (m, l) are polled in one loop, so the
  // merge starts one round trip after the last state is published.
  const int c = t & (kHeadDim - 1), g = t >> 7;
  constexpr int kB = 16;
  uint64_t ov[kB];
  uint32_t pend = 0;
#pragma unroll
  for (int r = 0; r < kB; ++r)
    if (g + 4 * r < total) pend |= 1u << r;
  float mt = kNegInf;
  for (int it = 0; it < kFSpin; ++it) {
#pragma unroll
    for (int r = 0; r < kB; ++r)
      if ((pend >> r) & 1u) ov[r] = get_tag(PRR_ELEM(g + 4 * r, c));
    bool ml_ok = true;
    for (int i = t; i < total; i += kFT) {
      const uint64_t vm = get_tag(PRR_ELEM(i, kHeadDim)), vl = get_tag(PRR_ELEM(i, kHeadDim + 1));
      ml_ok = ml_ok && tag_is(vm, a.epoch) && tag_is(vl, a.epoch);
      L.m[i] = __uint_as_float((uint32_t)vm);
      L.w[i] = __uint_as_float((uint32_t)vl);
    }
#pragma unroll
    for (int r = 0; r < kB; ++r)
      if (((pend >> r) & 1u) && tag_is(ov[r], a.epoch)) pend &= ~(1u << r);
    if (!pend && ml_ok) break;
    __builtin_amdgcn_s_sleep(1);
    if (it == kFSpin - 1) atomicOr(a.flags, kFlagSpinTimeout);
  }
  for (int i = t; i < total; i += kFT)
    if (L.w[i] > 0.0f) mt = fmaxf(mt, L.m[i]);
  mt = wave_max(mt);
  if (lane == 0) L.red[0][w] = mt;
  __syncthreads();
  float M = kNegInf;
#pragma unroll
  for (int i = 0; i < kFW; ++i) M = fmaxf(M, L.red[0][i]);
  float lsum_part = 0.0f;
  for (int i = t; i < total; i += kFT) {
    const float li = L.w[i];
    const float wi = li > 0.0f ? li * exp2f((L.m[i] - M) * kLog2e) : 0.0f;
    lsum_part += wi;
    L.w[i] = wi;
  }
  lsum_part = wave_sum(lsum_part);
  if (lane == 0) L.red[1][w] = lsum_part;
  __syncthreads();
  float Lsum = 0.0f;
#pragma unroll
  for (int i = 0; i < kFW; ++i) Lsum += L.red[1][i];

  float acc = 0.0f;
  for (int b0 = 0; b0 < total; b0 += 4 * kB) {
#pragma unroll
    for (int r = 0; r < kB; ++r) {
      const int i = b0 + g + 4 * r;
      if (b0 > 0 && i < total) ov[r] = get_tag(PRR_ELEM(i, c));
    }
#pragma unroll
    for (int r = 0; r < kB; ++r) {
      const int i = b0 + g + 4 * r;
      if (i < total) acc += L.w[i] * __uint_as_float(tagged(ov[r], PRR_ELEM(i, c), a.epoch, a.flags));
    }
  }
  L.acc[g][c] = acc;
  __syncthreads();
  if (g == 0) {
    const float sum = (L.acc[0][c] + L.acc[1][c]) + (L.acc[2][c] + L.acc[3][c]);
    const float o = Lsum > 0.0f ? sum / Lsum : 0.0f;
    const size_t row = (size_t)h * G + qn;
    a.out_o32[row * kHeadDim + c] = o;
    if (a.out_o) static_cast<uint16_t*>(a.out_o)[row * kHeadDim + c] = (uint16_t)f2h_rne<BF16>(o);
    if (c == 0) {
      a.out_m[row] = Lsum > 0.0f ? M : kNegInf;
      a.out_l[row] = Lsum;
    }
  }
#undef PRR_ELEM
}

// ------------------------------------------------------------------------ kernel

template <bool BF16, int PS, int NPW>
__global__ __launch_bounds__(kFT) void fused_step_kernel(const FusedLaunch a) {
  __shared__ FLds U;
  int b = blockIdx.x;
  const int H = a.num_kv_heads;
  if (b < H * a.n_score) {
    role_score<BF16>(a, b / a.n_score, b % a.n_score, U.score);
    return;
  }
  b -= H * a.n_score;
  if (b < H) {
    switch (sel2_j(a.num_pages, kFT)) {
      case 1: role_select<BF16, PS, 1>(a, b, U); break;
      case 2: role_select<BF16, PS, 2>(a, b, U); break;
      case 4: role_select<BF16, PS, 4>(a, b, U); break;
      case 8: role_select<BF16, PS, 8>(a, b, U); break;
      default: role_select<BF16, PS, 16>(a, b, U); break;
    }
    return;
  }
  b -= H;
  if (a.schedule != 0) {
    if (b < H) {
      switch (sel2_j(a.num_pages, kFT)) {
        case 1: role_predict<1>(a, b, U); break;
        case 2: role_predict<2>(a, b, U); break;
        case 4: role_predict<4>(a, b, U); break;
        case 8: role_predict<8>(a, b, U); break;
        default: role_predict<16>(a, b, U); break;
      }
      return;
    }
    b -= H;
  }
  if (a.schedule == 2) return;
  if (a.schedule == 1) {
    if (b < H * a.n_spec) {
      role_spec<BF16, PS, NPW>(a, b / a.n_spec, b % a.n_spec, U);
      return;
    }
    b -= H * a.n_spec;
  }
  if (b < H * a.n_miss) {
    role_miss<BF16, PS, NPW>(a, b / a.n_miss, b % a.n_miss, U);
    return;
  }
  b -= H * a.n_miss;
  if (b < H * a.group) role_merge<BF16>(a, b / a.group, b % a.group, U.merge);
}

template <typename K>
hipError_t launch_k(K kernel, int grid, const FusedLaunch& a, hipStream_t stream) {
  void* args[] = {const_cast<FusedLaunch*>(&a)};
  return hipLaunchKernel(reinterpret_cast<const void*>(kernel), dim3(grid), dim3(kFT), args, 0, stream);
}

}  // namespace

int fused_grid(const FusedLaunch& a) {
  const int H = a.num_kv_heads;
  int per = a.n_score + 1;
  if (a.schedule != 0) per += 1;
  if (a.schedule == 1) per += a.n_spec;
  if (a.schedule != 2) per += a.n_miss + a.group;
  return H * per;
}

hipError_t launch_fused(const FusedLaunch& a, bool bf16, int page_size, hipStream_t stream) {
  const int grid = fused_grid(a);
  const int npw = (a.chunk + kFW - 1) / kFW;
  if (page_size == 16) {
    if (npw <= 1)
      return bf16 ? launch_k(fused_step_kernel<true, 16, 1>, grid, a, stream)
                  : launch_k(fused_step_kernel<false, 16, 1>, grid, a, stream);
    return bf16 ? launch_k(fused_step_kernel<true, 16, 2>, grid, a, stream)
                : launch_k(fused_step_kernel<false, 16, 2>, grid, a, stream);
  }
  return bf16 ? launch_k(fused_step_kernel<true, 64, 1>, grid, a, stream)
              : launch_k(fused_step_kernel<false, 64, 1>, grid, a, stream);
}

}  // namespace prr
