// gfx950 (CDNA4) kernels of the speculate-reuse-repair decode path.
//
//   meta_minmax / meta_mean   page metadata (Appendix A.1; block means)
//   score_topk                GQA criticality of every page + top-K select, one launch:
//                             every workgroup scores a slice of pages, the last one to
//                             finish (per KV head) selects in LDS
//   predict                   EMA update and prediction (Section 4.1, Eqs. (2)-(3)) + top-|P|
//   spec_attn                 split-K flash-decode over a page list (Section 4.3)
//   repair                    set difference, missed / unmerge work units, merge
//                             (Section 4.3, Eqs. (6)-(8)), one launch
//   merge_states              stand-alone merge of partial states
//
// Wave64 throughout.  Attention uses MFMA: q.k^T as 16x16x32 bf16/f16 tiles (16 tokens x
// 16 query heads, contraction over the 128 channels), p.V by pv_tile (prr_device.h:
// bfloat16 MFMAs with the weights split into two bfloat16 terms, or fp32 MFMAs for float16).
#include <map>
#include <mutex>

#include "prr_device.h"
#include "prr_launch.h"
#include "prr_select.h"

namespace prr {


// =====================================================================================
// epoch of captured fused steps: one thread advances the word (skipping 0)
// =====================================================================================

__global__ void epoch_advance_kernel(uint32_t* p) {
  if (threadIdx.x == 0) {
    const uint32_t v = *p + 1u;
    *p = v == 0u ? 1u : v;
  }
}

hipError_t launch_epoch_advance(uint32_t* epoch_dev, hipStream_t stream) {
  void* args[] = {&epoch_dev};
  return hipLaunchKernel((const void*)epoch_advance_kernel, dim3(1), dim3(64), args, 0, stream);
}

// =====================================================================================
// workspace fill
// =====================================================================================

// An empty kernel: the launch floor of a grid of a given shape.
__global__ void empty_kernel() {}

hipError_t launch_empty(int grid, int threads, hipStream_t stream) {
  return hipLaunchKernel((const void*)empty_kernel, dim3(grid), dim3(threads), nullptr, 0, stream);
}

// Read-stream rate: every 16-byte word of the buffer read once (eight loads in flight
// per thread, consecutive lanes on consecutive words), folded into one word per
// workgroup so that the loads stay live.
__global__ void __launch_bounds__(256) read_stream_kernel(const u32x4_t* __restrict__ p, size_t n16,
                                                          uint32_t* __restrict__ sink) {
  constexpr int kU = 8;
  const size_t stride = (size_t)gridDim.x * 256;
  uint32_t acc = 0;
  size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  for (; i + (kU - 1) * stride < n16; i += kU * stride) {
    u32x4_t v[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) v[u] = __builtin_nontemporal_load(p + i + u * stride);
#pragma unroll
    for (int u = 0; u < kU; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (; i < n16; i += stride) {
    const u32x4_t v = p[i];
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  __shared__ uint32_t red[4];
  for (int o = 32; o > 0; o >>= 1) acc ^= __shfl_xor(acc, o);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) sink[blockIdx.x] = red[0] ^ red[1] ^ red[2] ^ red[3];
}

hipError_t launch_read_stream(const void* p, size_t bytes, uint32_t* sink, int grid, hipStream_t stream) {
  read_stream_kernel<<<grid, 256, 0, stream>>>(static_cast<const u32x4_t*>(p), bytes / 16, sink);
  return hipGetLastError();
}

__global__ void fill_zero_kernel(u32x4_t* __restrict__ p, size_t n16) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += stride) p[i] = u32x4_t{0, 0, 0, 0};
}

hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t stream) {
  const size_t n16 = bytes / 16;
  if (n16 == 0) return hipSuccess;
  size_t nb = (n16 + 255) / 256;
  const unsigned grid = (unsigned)(nb < 1024 ? nb : 1024);
  u32x4_t* ptr = reinterpret_cast<u32x4_t*>(p);
  size_t n = n16;
  void* args[] = {&ptr, &n};
  return hipLaunchKernel((const void*)fill_zero_kernel, dim3(grid), dim3(256), args, 0, stream);
}

// =====================================================================================
// page metadata
// =====================================================================================
// A wave takes kPages consecutive pages (two of 16 tokens, one from 32 on).  Lane l covers
// channels 8*(l%16) .. +8 of token rows l/16, l/16+4, .. of each page (16-byte loads, a wave
// load covers 4 full rows); the loads of all its pages are issued before any is reduced (8
// per lane in flight for 16- and 32-token pages, batches of 16 from 64 tokens on), then the
// four row groups are combined with cross-lane shuffles.  K is read once, with non-temporal
// loads.  Measured on the 128K GLM-shaped cache (18.5 us per layer with one 16-token page per
// wave and plain loads): two pages 18.0 us, four pages 20.0 us (22.2 with plain loads).
template <int PS>
struct MetaShape {
  static constexpr int kPages = PS >= 32 ? 1 : 32 / PS;  // pages per wave
  static constexpr int kRows = PS / 4;                   // row loads per lane and page
  static constexpr int kBatch = kRows < 16 ? kRows : 16; // row loads per lane issued together
};

// Pages per metadata workgroup (four waves).
template <int PS>
constexpr int meta_pages_per_block() {
  return 4 * MetaShape<PS>::kPages;
}

// The pages of this wave: source rows (lane's channels), valid tokens, and whether the
// page exists (in range, with a physical page inside the cache).
template <int PS>
__device__ __forceinline__ void meta_pages(const uint16_t* k, const int32_t* ptab, int num_tokens, int page_end,
                                           int max_pages, int h, int first, int cg,
                                           const uint16_t* (&src)[MetaShape<PS>::kPages],
                                           int (&valid)[MetaShape<PS>::kPages], bool (&ok)[MetaShape<PS>::kPages]) {
#pragma unroll
  for (int j = 0; j < MetaShape<PS>::kPages; ++j) {
    const int page = first + j;
    int phys = -1;
    if (page < page_end) phys = ptab ? ptab[page] : page;
    ok[j] = phys >= 0 && phys < max_pages;
    valid[j] = ok[j] ? min(PS, num_tokens - page * PS) : 0;
    src[j] = k + ((size_t)h * max_pages + (ok[j] ? phys : 0)) * PS * kHeadDim + cg * 8;
  }
}

template <bool BF16, int PS>
__global__ __launch_bounds__(256) void meta_minmax_kernel(const uint16_t* __restrict__ k, const int32_t* __restrict__ ptab,
                                                          int num_tokens, int page_begin, int page_end, int max_pages,
                                                          uint16_t* __restrict__ meta) {
  using S = MetaShape<PS>;
  const int h = blockIdx.y;
  const int lane = lane_id(), w = threadIdx.x / kWave;
  const int first = page_begin + (blockIdx.x * 4 + w) * S::kPages;
  if (first >= page_end) return;
  const int cg = lane & 15, rg = lane >> 4;
  const uint16_t* src[S::kPages];
  int valid[S::kPages];
  bool ok[S::kPages];
  meta_pages<PS>(k, ptab, num_tokens, page_end, max_pages, h, first, cg, src, valid, ok);
  float mn[S::kPages][8], mx[S::kPages][8];
#pragma unroll
  for (int j = 0; j < S::kPages; ++j) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      mn[j][e] = __builtin_inff();
      mx[j][e] = -__builtin_inff();
    }
  }
#pragma unroll
  for (int b = 0; b < S::kRows; b += S::kBatch) {
    u32x4_t v[S::kPages][S::kBatch];
#pragma unroll
    for (int j = 0; j < S::kPages; ++j) {
#pragma unroll
      for (int i = 0; i < S::kBatch; ++i) {
        const int r = (b + i) * 4 + rg;
        v[j][i] = r < valid[j] ? __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(src[j] + (size_t)r * kHeadDim))
                               : u32x4_t{0, 0, 0, 0};
      }
    }
#pragma unroll
    for (int j = 0; j < S::kPages; ++j) {
#pragma unroll
      for (int i = 0; i < S::kBatch; ++i) {
        if ((b + i) * 4 + rg < valid[j]) {
          const uint4 u = make_uint4(v[j][i].x, v[j][i].y, v[j][i].z, v[j][i].w);
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float f = u4_elem<BF16>(u, e);
            mn[j][e] = fminf(mn[j][e], f);
            mx[j][e] = fmaxf(mx[j][e], f);
          }
        }
      }
    }
  }
#pragma unroll
  for (int j = 0; j < S::kPages; ++j) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      mn[j][e] = fminf(mn[j][e], __shfl_xor(mn[j][e], 16));
      mn[j][e] = fminf(mn[j][e], __shfl_xor(mn[j][e], 32));
      mx[j][e] = fmaxf(mx[j][e], __shfl_xor(mx[j][e], 16));
      mx[j][e] = fmaxf(mx[j][e], __shfl_xor(mx[j][e], 32));
    }
    if (ok[j] && rg < 2) {
      const float* x = rg == 0 ? mn[j] : mx[j];
      uint4 o;
      o.x = f2h_exact<BF16>(x[0]) | (f2h_exact<BF16>(x[1]) << 16);
      o.y = f2h_exact<BF16>(x[2]) | (f2h_exact<BF16>(x[3]) << 16);
      o.z = f2h_exact<BF16>(x[4]) | (f2h_exact<BF16>(x[5]) << 16);
      o.w = f2h_exact<BF16>(x[6]) | (f2h_exact<BF16>(x[7]) << 16);
      *reinterpret_cast<uint4*>(meta + (((size_t)h * max_pages + first + j) * 2 + rg) * kHeadDim + cg * 8) = o;
    }
  }
}

template <bool BF16, int PS>
__global__ __launch_bounds__(256) void meta_mean_kernel(const uint16_t* __restrict__ k, const int32_t* __restrict__ ptab,
                                                        int num_tokens, int page_begin, int page_end, int max_pages,
                                                        float* __restrict__ meta) {
  using S = MetaShape<PS>;
  const int h = blockIdx.y;
  const int lane = lane_id(), w = threadIdx.x / kWave;
  const int first = page_begin + (blockIdx.x * 4 + w) * S::kPages;
  if (first >= page_end) return;
  const int cg = lane & 15, rg = lane >> 4;
  const uint16_t* src[S::kPages];
  int valid[S::kPages];
  bool ok[S::kPages];
  meta_pages<PS>(k, ptab, num_tokens, page_end, max_pages, h, first, cg, src, valid, ok);
  float sm[S::kPages][8];
#pragma unroll
  for (int j = 0; j < S::kPages; ++j) {
#pragma unroll
    for (int e = 0; e < 8; ++e) sm[j][e] = 0.0f;
  }
#pragma unroll
  for (int b = 0; b < S::kRows; b += S::kBatch) {
    u32x4_t v[S::kPages][S::kBatch];
#pragma unroll
    for (int j = 0; j < S::kPages; ++j) {
#pragma unroll
      for (int i = 0; i < S::kBatch; ++i) {
        const int r = (b + i) * 4 + rg;
        v[j][i] = r < valid[j] ? __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(src[j] + (size_t)r * kHeadDim))
                               : u32x4_t{0, 0, 0, 0};
      }
    }
#pragma unroll
    for (int j = 0; j < S::kPages; ++j) {
#pragma unroll
      for (int i = 0; i < S::kBatch; ++i) {
        if ((b + i) * 4 + rg < valid[j]) {
          const uint4 u = make_uint4(v[j][i].x, v[j][i].y, v[j][i].z, v[j][i].w);
#pragma unroll
          for (int e = 0; e < 8; ++e) sm[j][e] += u4_elem<BF16>(u, e);
        }
      }
    }
  }
#pragma unroll
  for (int j = 0; j < S::kPages; ++j) {
    const float inv = 1.0f / (float)valid[j];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      sm[j][e] += __shfl_xor(sm[j][e], 16);
      sm[j][e] += __shfl_xor(sm[j][e], 32);
    }
    if (ok[j] && rg == 0) {
      float4* dst = reinterpret_cast<float4*>(meta + ((size_t)h * max_pages + first + j) * kHeadDim + cg * 8);
      dst[0] = make_float4(sm[j][0] * inv, sm[j][1] * inv, sm[j][2] * inv, sm[j][3] * inv);
      dst[1] = make_float4(sm[j][4] * inv, sm[j][5] * inv, sm[j][6] * inv, sm[j][7] * inv);
    }
  }
}

// The instance of a kernel template for a page size (16, 32, 64, 128 or 256 tokens), or
// NULL for another size (the C ABI admits only these).
template <typename K>
const void* by_page_size(int ps) {
  switch (ps) {
    case 16: return K::template get<16>();
    case 32: return K::template get<32>();
    case 64: return K::template get<64>();
    case 128: return K::template get<128>();
    case 256: return K::template get<256>();
    default: return nullptr;
  }
}

template <bool BF16>
struct MetaMeanK {
  template <int PS>
  static const void* get() { return (const void*)meta_mean_kernel<BF16, PS>; }
};
template <bool BF16>
struct MetaMinmaxK {
  template <int PS>
  static const void* get() { return (const void*)meta_minmax_kernel<BF16, PS>; }
};

hipError_t launch_meta(const MetaLaunch& a, hipStream_t stream) {
  const int np = a.page_end - a.page_begin;
  if (np <= 0) return hipSuccess;
  int ppb = 0;  // pages per workgroup
  switch (a.page_size) {
    case 16: ppb = meta_pages_per_block<16>(); break;
    case 32: ppb = meta_pages_per_block<32>(); break;
    case 64: ppb = meta_pages_per_block<64>(); break;
    case 128: ppb = meta_pages_per_block<128>(); break;
    case 256: ppb = meta_pages_per_block<256>(); break;
    default: return hipErrorInvalidValue;
  }
  dim3 grid((np + ppb - 1) / ppb, a.num_kv_heads);
  const uint16_t* k = static_cast<const uint16_t*>(a.k_cache);
  const int32_t* ptab = a.page_table;
  int nt = a.num_tokens, pb = a.page_begin, pe = a.page_end, mp = a.max_pages;
  void* meta = a.meta;
  void* args[] = {&k, &ptab, &nt, &pb, &pe, &mp, &meta};
  const void* f = a.meta_mean ? (a.bf16 ? by_page_size<MetaMeanK<true>>(a.page_size) : by_page_size<MetaMeanK<false>>(a.page_size))
                              : (a.bf16 ? by_page_size<MetaMinmaxK<true>>(a.page_size)
                                        : by_page_size<MetaMinmaxK<false>>(a.page_size));
  if (!f) return hipErrorInvalidValue;
  return hipLaunchKernel(f, grid, dim3(256), args, 0, stream);
}

// =====================================================================================
// block top-K select (shared by score_topk and predict)
// =====================================================================================
// 1024 threads; thread (wave w, lane) owns pages w*J*64 + j*64 + lane, j < J, with their
// keys in registers, so that (w, j, lane) is ascending page order.  Candidates have their
// bit set in `cand`, pages in `force` are always selected.
//
// All pages of a KV head are candidates here, so their keys span the whole range of the
// scores (negative and positive), and radix bins over the key bits put most keys into a
// few bins, whose LDS atomics then serialise.  The first pass therefore bins the values
// linearly between the smallest and the largest candidate (a non-decreasing map, so a
// higher bin holds only larger values); the key-space radix select of prr_select.h then
// ranks the keys of the one bin that holds rank kextra.  Keys of NaN or infinite values
// fall back to the key-space select.  The selection is emitted in ascending page order
// by ballot compaction.

constexpr int kSelThreads = 1024;

struct __align__(16) SelectScratch {
  Sel2Lds sel;
  uint32_t forceb[PRR_MAX_PAGES_DEV / 32];
  int wcnt[kSelThreads / kWave];  // selected pages per wave
};

__host__ __device__ inline int select_j(int n) { return sel2_j(n, kSelThreads); }

// the float whose score_key is k
__device__ __forceinline__ float key_value(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

template <int J>
__device__ __forceinline__ void select_topk_regs(const uint32_t (&key)[J], uint64_t cand, uint64_t force, int kextra,
                                                 int32_t* __restrict__ out, int cap, int32_t* __restrict__ out_count,
                                                 SelectScratch& ss) {
  constexpr int NT = kSelThreads, NW = NT / kWave;
  Sel2Lds& S = ss.sel;
  const int t = threadIdx.x, lane = lane_id(), w = t / kWave;
  int page[J];
#pragma unroll
  for (int j = 0; j < J; ++j) page[j] = sel2_page<J>(j);

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
  const float vlo = key_value(lo), span = key_value(hi) - vlo;
  const float scale = (float)kSel2Bins / span;

  // S.red is next written by the list compaction (after the barriers of the passes below)
  // or, on the key-space path, right at its start, hence the barrier there
  uint64_t in;
  int eq_cut = -1;
  if (kextra <= 0 || cnt == 0) {
    in = force;
  } else if (kextra >= cnt) {
    in = cand | force;
  } else if (!(span > 0.0f) || !__builtin_isfinite(span) || !__builtin_isfinite(scale)) {
    __syncthreads();
    const SelThreshold th = sel2_threshold<NT, J>(key, cand, kextra, S);
    in = sel2_membership<NT, J>(key, page, cand, force, th, &eq_cut, S);
  } else {
    int bin[J];
#pragma unroll
    for (int j = 0; j < J; ++j) {
      bin[j] = min(kSel2Bins - 1, (int)((key_value(key[j]) - vlo) * scale));
      if ((cand >> j) & 1ull) atomicAdd(&S.hist[0][bin[j]], 1u);
    }
    __syncthreads();
    if (w == 0) {
      // lane l owns bins [2048 - 32(l+1), 2048 - 32l); the lane holding rank kextra, then
      // its bin (the scan of prr_select.h's first pass)
      const int base = kSel2Bins - 32 * (lane + 1);
      const uint4* hb = reinterpret_cast<const uint4*>(S.hist[0] + base);
      int sum = 0;
#pragma unroll
      for (int v = 0; v < 8; ++v) {
        const uint4 x = hb[v];
        sum += (int)(x.x + x.y + x.z + x.w);
      }
      const int incl = wave_inclusive_scan(sum);
      const int excl = incl - sum;
      const uint64_t hit = __ballot(excl < kextra && kextra <= incl);
      const int ls = __builtin_amdgcn_readfirstlane(__ffsll((long long)hit) - 1);
      const int ex = __builtin_amdgcn_readlane(excl, ls);
      const int lbase = kSel2Bins - 32 * (ls + 1);
      const int cj = lane < 32 ? (int)S.hist[0][lbase + 31 - lane] : 0;
      const int cinc = wave_inclusive_scan(cj);
      const uint64_t hit2 = __ballot(lane < 32 && ex + cinc >= kextra);
      const int js = __builtin_amdgcn_readfirstlane(__ffsll((long long)hit2) - 1);
      if (lane == js) {
        S.res[0] = lbase + 31 - js;
        S.res[1] = ex + cinc - cj;
        S.res[2] = cj;
      }
    }
    __syncthreads();
    const int bstar = S.res[0], above = S.res[1], cbin = S.res[2];
    const int rank = kextra - above;  // of the threshold among the boundary bin's keys
    uint64_t inbin = 0, upper = 0;
#pragma unroll
    for (int j = 0; j < J; ++j) {
      if ((cand >> j) & 1ull) {
        if (bin[j] == bstar) inbin |= 1ull << j;
        if (bin[j] > bstar) upper |= 1ull << j;
      }
    }
    // every value in a higher bin is larger than every value of the boundary bin, and
    // keys equal to the threshold share its bin, so the tie cut is the boundary bin's
    SelThreshold th;
    if (cbin <= kSel2Small) {
      // the few keys of the boundary bin, ranked directly by one wave
      const int mine = __popcll(inbin);
      if (mine) {
        int slot = atomicAdd(&S.nsmall, mine);
#pragma unroll
        for (int j = 0; j < J; ++j)
          if ((inbin >> j) & 1ull) S.small[slot++] = key[j];
      }
      __syncthreads();
      if (w == 0) {
        const uint32_t kx = S.small[lane < cbin ? lane : 0];
        int gt = 0, ge = 0;
        for (int x = 0; x < cbin; ++x) {
          const uint32_t ky = (uint32_t)__builtin_amdgcn_readlane((int)kx, x);
          gt += ky > kx ? 1 : 0;
          ge += ky >= kx ? 1 : 0;
        }
        const uint64_t hit = __ballot(lane < cbin && gt < rank && rank <= ge);
        const int ls = __builtin_amdgcn_readfirstlane(__ffsll((long long)hit) - 1);
        if (lane == ls) {
          S.res[3] = (int)kx;
          S.res[4] = rank - gt;
          S.res[5] = ge - gt;
        }
      }
      __syncthreads();
      th.mode = 2;
      th.T = (uint32_t)S.res[3];
      th.need_eq = S.res[4];
      th.eq_total = S.res[5];
    } else {
      __syncthreads();  // S.res and the histogram are reused by the select of the boundary bin
      th = sel2_threshold<NT, J>(key, inbin, rank, S);
    }
    in = sel2_membership<NT, J>(key, page, inbin, force | upper, th, &eq_cut, S);
  }
  // ascending page order: the waves before this one, then ballot ranks within the wave
  // (ss.wcnt is not read before this point, so one barrier suffices)
  const int c = wave_isum(__popcll(in));
  if (lane == 0) ss.wcnt[w] = c;
  __syncthreads();
  int run = 0, total = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    const int ci = ss.wcnt[i];
    run += i < w ? ci : 0;
    total += ci;
  }
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const bool sel = (in >> j) & 1ull;
    const uint64_t bm = __ballot(sel);
    if (sel) {
      const int pos = run + lanes_below(bm);
      if (pos < cap) out[pos] = page[j];
    }
    run += __popcll(bm);
  }
  if (t == 0) *out_count = min(total, cap);
}

// Forced pages as a bitmap in LDS; returns this thread's J-bit mask.
template <int J>
__device__ __forceinline__ uint64_t forced_mask(const int32_t* forced, int n_forced, int n, uint32_t* forceb) {
  if (n_forced == 0) return 0;
  const int nw = (n + 31) / 32;
  for (int i = threadIdx.x; i < nw; i += kSelThreads) forceb[i] = 0u;
  __syncthreads();
  if ((int)threadIdx.x < n_forced) {
    const int p = forced[threadIdx.x];
    atomicOr(&forceb[p >> 5], 1u << (p & 31));
  }
  __syncthreads();
  uint64_t m = 0;
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int pj = sel2_page<J>(j);
    const int p = min(pj, n - 1);
    if (pj < n && ((forceb[p >> 5] >> (p & 31)) & 1u)) m |= 1ull << j;
  }
  return m;
}

// =====================================================================================
// score + top-K
// =====================================================================================
// grid (ceil(num_pages / 64), Hkv), 1024 threads.  Wave w of a workgroup scores pages
// base + w*4 + (lane/16); lane%16 covers channels 8*(lane%16)..+8.
constexpr int kScorePagesPerWg = 64;

// The selecting workgroup: this KV head's scores (published by every workgroup with
// device-coherent stores) into registers, then the block select.
template <int J>
__device__ __forceinline__ void select_scores(const float* scores, int n, const ScoreLaunch& a, int h,
                                              SelectScratch& ss) {
  uint32_t key[J];
  uint64_t cand = 0;
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int p = sel2_page<J>(j);
    key[j] = score_key(ld_dev(&scores[min(p, n - 1)]));
    if (p < n) cand |= 1ull << j;
  }
  const uint64_t force = forced_mask<J>(a.forced, a.n_forced, n, ss.forceb);
  cand &= ~force;
  select_topk_regs<J>(key, cand, force, a.kextra, a.selected + (size_t)h * a.cap, a.cap, a.selected_count + h, ss);
}

template <bool BF16, bool MEAN>
__global__ __launch_bounds__(1024) void score_topk_kernel(const ScoreLaunch a) {
  __shared__ SelectScratch ss;
  __shared__ float qbar[kHeadDim];
  __shared__ float qpart[16][kHeadDim];
  __shared__ int s_last;
  const int h = blockIdx.y;
  const int t = threadIdx.x, lane = lane_id(), w = t / kWave;
  const int G = a.group;
  const uint16_t* q = static_cast<const uint16_t*>(a.q);

  {
    // thread t < 16G loads 8 channels of query head t/16 of this group (one 16-byte load);
    // the group mean is then summed in head order from LDS
    const int g = t >> 4, c8 = (t & 15) * 8;
    if (g < G) {
      const uint4 v = *reinterpret_cast<const uint4*>(q + (size_t)(h * G + g) * kHeadDim + c8);
#pragma unroll
      for (int e = 0; e < 8; ++e) qpart[g][c8 + e] = u4_elem<BF16>(v, e);
    }
    __syncthreads();
    if (t < kHeadDim) {
      float s = 0.0f;
      for (int gg = 0; gg < G; ++gg) s += qpart[gg][t];
      qbar[t] = s / (float)G;
    }
    __syncthreads();
  }

  const int cg = lane & 15, pi = lane >> 4;
  float qb[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) qb[e] = qbar[cg * 8 + e];

  const int page = blockIdx.x * kScorePagesPerWg + w * 4 + pi;
  float* scores = a.scores + (size_t)h * a.max_pages;
  float s = 0.0f;
  if constexpr (!MEAN) {
    if (page < a.num_pages) {
      const uint16_t* row = static_cast<const uint16_t*>(a.meta) + ((size_t)h * a.max_pages + page) * 2 * kHeadDim + cg * 8;
      const uint4 mn = *reinterpret_cast<const uint4*>(row);
      const uint4 mx = *reinterpret_cast<const uint4*>(row + kHeadDim);
#pragma unroll
      for (int e = 0; e < 8; ++e) s += fmaxf(qb[e] * u4_elem<BF16>(mn, e), qb[e] * u4_elem<BF16>(mx, e));
    }
  } else {
    if (page < a.num_pages) {
      const float4* row = reinterpret_cast<const float4*>(static_cast<const float*>(a.meta) +
                                                          ((size_t)h * a.max_pages + page) * kHeadDim + cg * 8);
      const float4 m0 = row[0], m1 = row[1];
      s = qb[0] * m0.x;
      s += qb[1] * m0.y;
      s += qb[2] * m0.z;
      s += qb[3] * m0.w;
      s += qb[4] * m1.x;
      s += qb[5] * m1.y;
      s += qb[6] * m1.z;
      s += qb[7] * m1.w;
    }
  }
  s = sum16(s);
  if (cg == 0 && page < a.num_pages) st_dev(&scores[page], s);

  // the last workgroup of this KV head selects: scores are published with device-coherent
  // stores, completed before the counter is bumped, and read back the same way
  stores_complete();
  __syncthreads();
  if (t == 0) {
    const uint32_t old = counter_add(&a.counters[h], 1u);
    s_last = (old == (uint32_t)(gridDim.x - 1));
  }
  __syncthreads();
  if (!s_last) return;

  const int n = a.num_pages;
  switch (select_j(n)) {
    case 1: select_scores<1>(scores, n, a, h, ss); break;
    case 2: select_scores<2>(scores, n, a, h, ss); break;
    case 4: select_scores<4>(scores, n, a, h, ss); break;
    case 8: select_scores<8>(scores, n, a, h, ss); break;
    default: select_scores<16>(scores, n, a, h, ss); break;
  }
  if (t == 0) atomicExch(&a.counters[h], 0u);
}

// =====================================================================================
// EMA predictor
// =====================================================================================

template <int J>
__device__ __forceinline__ void predict_head(const PredictLaunch& a, int h, SelectScratch& ss) {
  const int lane = lane_id();
  const int n = a.num_pages;
  const int nwmax = (a.max_pages + 31) / 32;
  float* level = a.level + (size_t)h * a.max_pages;
  float* trend = a.trend + (size_t)h * a.max_pages;
  uint32_t* bits = a.init_bits + (size_t)h * nwmax;
  const float* scores = a.scores ? a.scores + (size_t)h * a.max_pages : nullptr;
  // all loads first (clamped addresses; a wave covers 64 consecutive pages = two bit words per j)
  float lv[J], tv[J], sc[J];
  uint32_t bw[J];
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int p = min(sel2_page<J>(j), n - 1);
    lv[j] = level[p];
    tv[j] = trend[p];
    sc[j] = scores ? scores[p] : 0.0f;
    bw[j] = bits[p >> 5];
  }
  uint32_t key[J];
  uint64_t cand = 0;
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int p = sel2_page<J>(j);
    const bool inr = p < n;
    bool has = inr && ((bw[j] >> (p & 31)) & 1u);
    float l = lv[j], v = tv[j];
    if (inr && scores) {
      const float s = sc[j];
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
    if (has) cand |= 1ull << j;
    const uint64_t hm = __ballot(has);
    const uint64_t vm = __ballot(inr);
    if (scores && (lane == 0 || lane == 32)) {
      const uint32_t hbits = (uint32_t)(lane == 0 ? hm : (hm >> 32));
      const uint32_t vbits = (uint32_t)(lane == 0 ? vm : (vm >> 32));
      if (vbits) bits[p >> 5] = (bw[j] & ~vbits) | hbits;
    }
  }
  const uint64_t force = forced_mask<J>(a.forced, a.n_forced, n, ss.forceb);
  cand &= ~force;
  select_topk_regs<J>(key, cand, force, a.kextra, a.predicted + (size_t)h * a.cap, a.cap, a.predicted_count + h,
                      ss);
}

__global__ __launch_bounds__(1024) void predict_kernel(const PredictLaunch a) {
  __shared__ SelectScratch ss;
  const int h = blockIdx.x;
  switch (select_j(a.num_pages)) {
    case 1: predict_head<1>(a, h, ss); break;
    case 2: predict_head<2>(a, h, ss); break;
    case 4: predict_head<4>(a, h, ss); break;
    case 8: predict_head<8>(a, h, ss); break;
    default: predict_head<16>(a, h, ss); break;
  }
}

// =====================================================================================
// attention over a short page list (one workgroup, four waves)
// =====================================================================================
// Wave w takes list entries w, w+4, w+8, w+12 (a list holds at most 16 tiles of 16 tokens
// per wave group, i.e. chunk_pages * page_size / 16 <= 16) and runs an online softmax
// over their 16-token tiles; the four wave states are merged in LDS.
//
// q.k^T per tile: S^T (16 tokens x 16 heads) = K (16 x 128) . Q^T (128 x 16) as four
// 16x16x32 MFMAs.  The contraction index is permuted so that each lane reads 64
// contiguous bytes of its key row: for k-step s, lane 16j+r supplies channels
// 32j+8s .. +8 of token r (A operand) and lane 16j+n channels 32j+8s .. +8 of query head n
// (B operand).  The result gives lane 16j+n the logits of tokens 4j..4j+3 for head n.
//
// p.V per tile, transposed: O^T (128 channels x 16 heads) += V^T . P^T by pv_tile
// (prr_device.h): lane 16j+m supplies channel 8m+cb of V rows 4j..4j+3 (from one 16-byte
// row load per row) and the weights of head m for tokens 4j..4j+3 (its own logit
// registers).  Accumulator cb, register i of lane 16j+n then holds O[head n][32j + 8i + cb]:
// each lane owns 32 contiguous channels of the same head whose logits it holds, so the
// online rescale is lane-local.

struct AttnCtx {
  const uint16_t* q;  // q + h*G*128
  const uint16_t* k;  // k_cache + h*max_pages*PS*128
  const uint16_t* v;
  const int32_t* ptab;
  int max_pages, num_pages, num_tokens, G;
};

constexpr int kOPad = kHeadDim + 4;  // LDS row stride of a head's partial output

struct UnitLds {
  float wo[4][16][kOPad];
  float wm[4][16];
  float wl[4][16];
  float wpm[4][16];  // per-wave page maxima (pages of 128 and 256 tokens span several waves)
};

template <bool BF16>
__device__ __forceinline__ f32x4_t mfma_qk(const u32x4_t& a, const u32x4_t& b, f32x4_t c) {
  if constexpr (BF16) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b), c,
                                                   0, 0, 0);
  } else {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8_t, a), __builtin_bit_cast(f16x8_t, b), c, 0,
                                                  0, 0);
  }
}

// Result for thread t: head t/16, channels 8*(t%16)..+8: normalised o, m, l.
struct UnitResult {
  float o[8];
  float m, l;
};

// A unit is at most 16 tiles of 16 tokens, four per wave.  Pages of up to 64 tokens are
// whole to one wave (list entries w, w + 4, .. for wave w); a page of 128 or 256 tokens
// spans WPP = 2 or 4 waves (entry w / WPP, tiles 4 (w % WPP) .. + 3).
template <bool BF16, int PS>
__device__ void attend_unit(const AttnCtx& c, const int32_t* pages, int cnt, float* page_m_out, UnitLds& sm,
                            uint32_t* flags, UnitResult& res) {
  static_assert(PS == 16 || PS == 32 || PS == 64 || PS == 128 || PS == 256, "page size");
  constexpr int TPP = PS / 16;
  constexpr int NTL = 16 / 4;  // tiles per wave at most (16 tiles per unit)
  constexpr int NPW = TPP <= NTL ? NTL / TPP : 1;  // list entries per wave at most
  constexpr int WPP = TPP <= NTL ? 1 : TPP / NTL;  // waves per page
  constexpr int TW = TPP <= NTL ? NPW * TPP : NTL;  // tiles of one wave
  const float kNegInf = -__builtin_inff();
  const float scale = 0.08838834764831845f;  // 1/sqrt(128)
  const int t = threadIdx.x, lane = lane_id(), w = t / kWave;
  const int j = lane >> 4, n = lane & 15;
  const int G = c.G;

  u32x4_t qf[4];
  if (n < G) {
    const u32x4_t* src = reinterpret_cast<const u32x4_t*>(c.q + (size_t)n * kHeadDim + 32 * j);
#pragma unroll
    for (int s = 0; s < 4; ++s) qf[s] = src[s];
  } else {
#pragma unroll
    for (int s = 0; s < 4; ++s) qf[s] = u32x4_t{0, 0, 0, 0};
  }

  // list entries w, w+4, .. (or w / WPP): ids first, then page-table entries (wave-uniform values)
  const int wu = __builtin_amdgcn_readfirstlane(w);
  const int e0 = wu / WPP, tt0 = (wu % WPP) * NTL;  // (0 when a page is whole to a wave)
  int pg[NPW], ph[NPW];
#pragma unroll
  for (int kk = 0; kk < NPW; ++kk) {
    const int i = WPP == 1 ? wu + 4 * kk : e0;
    pg[kk] = i < cnt ? pages[i] : -1;
  }
#pragma unroll
  for (int kk = 0; kk < NPW; ++kk) {
    pg[kk] = __builtin_amdgcn_readfirstlane(pg[kk]);
    const bool in_list = (WPP == 1 ? wu + 4 * kk : e0) < cnt;
    const bool valid = pg[kk] >= 0 && pg[kk] < c.num_pages;
    if (in_list && !valid && flags && lane == 0) atomicOr(flags, kFlagBadListEntry);
    if (!valid) pg[kk] = -1;
  }
#pragma unroll
  for (int kk = 0; kk < NPW; ++kk) ph[kk] = (pg[kk] >= 0 && c.ptab) ? c.ptab[pg[kk]] : pg[kk];
  size_t off[NPW];
  int tok0[NPW];
  bool ok[NPW];
#pragma unroll
  for (int kk = 0; kk < NPW; ++kk) {
    const int phys = __builtin_amdgcn_readfirstlane(ph[kk]);
    ok[kk] = pg[kk] >= 0 && phys >= 0 && phys < c.max_pages;
    if (pg[kk] >= 0 && !ok[kk] && flags && lane == 0) atomicOr(flags, kFlagBadListEntry);
    off[kk] = ok[kk] ? (size_t)phys * PS * kHeadDim : 0;
    tok0[kk] = ok[kk] ? pg[kk] * PS : 0;
  }

  f32x4_t acc[8];
#pragma unroll
  for (int cb = 0; cb < 8; ++cb) acc[cb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m_run = kNegInf, l_run = 0.0f;

  // every tile of the wave is loaded up front (at most 4 tiles: 32 registers each)
  u32x4_t kf[NTL][4], vf[NTL][4];
#pragma unroll
  for (int f = 0; f < TW; ++f) {
    const int kk = WPP == 1 ? f / TPP : 0, tt = WPP == 1 ? f % TPP : tt0 + f;
    if (ok[kk]) {
      const uint16_t* kt = c.k + off[kk] + (size_t)tt * 16 * kHeadDim;
      const uint16_t* vt = c.v + off[kk] + (size_t)tt * 16 * kHeadDim;
      const u32x4_t* ks = reinterpret_cast<const u32x4_t*>(kt + (size_t)n * kHeadDim + 32 * j);
#pragma unroll
      for (int s = 0; s < 4; ++s) kf[f][s] = ks[s];
#pragma unroll
      for (int tg = 0; tg < 4; ++tg)
        vf[f][tg] = *reinterpret_cast<const u32x4_t*>(vt + (size_t)(4 * j + tg) * kHeadDim + 8 * n);
    }
  }

  float pm = kNegInf;  // max logit of the current page (this wave's tiles of it), head n
#pragma unroll
  for (int f = 0; f < TW; ++f) {
    const int kk = WPP == 1 ? f / TPP : 0, tt = WPP == 1 ? f % TPP : tt0 + f;
    if (!ok[kk]) continue;
    if (WPP == 1 && tt == 0) pm = kNegInf;
    f32x4_t st = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < 4; ++s) st = mfma_qk<BF16>(kf[f][s], qf[s], st);
    float sv[4];
    float mx = kNegInf;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int tok = tok0[kk] + tt * 16 + 4 * j + i;
      sv[i] = tok < c.num_tokens ? st[i] * scale : kNegInf;
      mx = fmaxf(mx, sv[i]);
    }
    mx = max_rows(mx);
    pm = fmaxf(pm, mx);
    const float mnew = fmaxf(m_run, mx);
    float alpha = 1.0f;
    float p[4] = {0.f, 0.f, 0.f, 0.f};
    if (mnew != kNegInf) {
      alpha = exp2f((m_run - mnew) * kLog2e);
#pragma unroll
      for (int i = 0; i < 4; ++i) p[i] = exp2f((sv[i] - mnew) * kLog2e);
    }
    const float ls = sum_rows((p[0] + p[1]) + (p[2] + p[3]));
    l_run = l_run * alpha + ls;
    m_run = mnew;
    if (tok0[kk] + PS > c.num_tokens) {
      // a partial last page: the values of tokens at or past num_tokens are zeroed, not
      // only weighted by 0 (0 x NaN or Inf from an unwritten cache tail would poison o)
#pragma unroll
      for (int tg = 0; tg < 4; ++tg)
        if (tok0[kk] + tt * 16 + 4 * j + tg >= c.num_tokens) vf[f][tg] = u32x4_t{0, 0, 0, 0};
    }
#pragma unroll
    for (int cb = 0; cb < 8; ++cb) {
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[cb][i] *= alpha;
    }
    pv_tile<BF16>(acc, vf[f], p);
    if (WPP == 1 && tt == TPP - 1 && page_m_out && j == 0 && n < G) page_m_out[(size_t)(w + 4 * kk) * G + n] = pm;
  }
  if constexpr (WPP > 1) {
    if (j == 0) sm.wpm[w][n] = pm;
  }

  // merge the four wave states: lane 16j+n holds channels 32j + 8i + cb of head n
  if (j == 0) {
    sm.wm[w][n] = m_run;
    sm.wl[w][n] = l_run;
  }
  float* row = &sm.wo[w][n][32 * j];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    *reinterpret_cast<float4*>(row + 8 * i) = make_float4(acc[0][i], acc[1][i], acc[2][i], acc[3][i]);
    *reinterpret_cast<float4*>(row + 8 * i + 4) = make_float4(acc[4][i], acc[5][i], acc[6][i], acc[7][i]);
  }
  __syncthreads();
  if constexpr (WPP > 1) {
    // page e's maximum over its waves (thread e * 16 + head)
    const int e = t >> 4, hd = t & 15;
    if (page_m_out && e < 4 / WPP && e < cnt && hd < G) {
      float m = kNegInf;
#pragma unroll
      for (int x = 0; x < WPP; ++x) m = fmaxf(m, sm.wpm[e * WPP + x][hd]);
      page_m_out[(size_t)e * G + hd] = m;
    }
  }
  const int hh = t >> 4, c0 = (t & 15) * 8;
  float mw[4], fw[4];
  float ms = kNegInf;
#pragma unroll
  for (int ww = 0; ww < 4; ++ww) {
    mw[ww] = sm.wm[ww][hh];
    if (sm.wl[ww][hh] > 0.0f) ms = fmaxf(ms, mw[ww]);
  }
  float L = 0.0f;
#pragma unroll
  for (int ww = 0; ww < 4; ++ww) {
    const float lw = sm.wl[ww][hh];
    fw[ww] = lw > 0.0f ? exp2f((mw[ww] - ms) * kLog2e) : 0.0f;
    L += lw * fw[ww];
  }
  const float inv = L > 0.0f ? 1.0f / L : 0.0f;
  float o[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ww = 0; ww < 4; ++ww) {
    const float4 a = *reinterpret_cast<const float4*>(&sm.wo[ww][hh][c0]);
    const float4 b = *reinterpret_cast<const float4*>(&sm.wo[ww][hh][c0 + 4]);
    o[0] += a.x * fw[ww];
    o[1] += a.y * fw[ww];
    o[2] += a.z * fw[ww];
    o[3] += a.w * fw[ww];
    o[4] += b.x * fw[ww];
    o[5] += b.y * fw[ww];
    o[6] += b.z * fw[ww];
    o[7] += b.w * fw[ww];
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) res.o[e] = o[e] * inv;
  res.m = L > 0.0f ? ms : kNegInf;
  res.l = L;
  __syncthreads();
}

template <bool BF16, int PS>
__global__ __launch_bounds__(256) void spec_attn_kernel(const SpecLaunch a) {
  __shared__ UnitLds sm;
  __shared__ int32_t ids[16];
  const int c = blockIdx.x, h = blockIdx.y;
  const int start = c * a.chunk;
  // the chunk's page ids (at most 16) are loaded together with the count, clamped to the
  // capacity, so that the count costs no round trip of its own
  int id = -1;
  if ((int)threadIdx.x < a.chunk) id = a.pages[(size_t)h * a.cap + min(start + (int)threadIdx.x, a.cap - 1)];
  const int total = min(max(a.page_count[h], 0), a.cap);
  if (start >= total) return;
  const int cnt = min(a.chunk, total - start);
  if ((int)threadIdx.x < a.chunk) ids[threadIdx.x] = id;
  __syncthreads();
  const int G = a.group;
  AttnCtx ctx;
  ctx.q = static_cast<const uint16_t*>(a.q) + (size_t)h * G * kHeadDim;
  ctx.k = static_cast<const uint16_t*>(a.k_cache) + (size_t)h * a.max_pages * a.page_size * kHeadDim;
  ctx.v = static_cast<const uint16_t*>(a.v_cache) + (size_t)h * a.max_pages * a.page_size * kHeadDim;
  ctx.ptab = a.page_table;
  ctx.max_pages = a.max_pages;
  ctx.num_pages = a.num_pages;
  ctx.num_tokens = a.num_tokens;
  ctx.G = G;
  UnitResult r;
  float* pmo = a.page_m ? a.page_m + ((size_t)h * a.cap + start) * G : nullptr;
  attend_unit<BF16, PS>(ctx, ids, cnt, pmo, sm, nullptr, r);
  const int t = threadIdx.x, hh = t >> 4, c0 = (t & 15) * 8;
  if (hh < G) {
    const size_t row = ((size_t)h * a.nchunks + c) * G + hh;
    float4* dst = reinterpret_cast<float4*>(a.part_o + row * kHeadDim + c0);
    dst[0] = make_float4(r.o[0], r.o[1], r.o[2], r.o[3]);
    dst[1] = make_float4(r.o[4], r.o[5], r.o[6], r.o[7]);
    if ((t & 15) == 0) {
      a.part_m[row] = r.m;
      a.part_l[row] = r.l;
    }
  }
}

// =====================================================================================
// repair
// =====================================================================================
// Grid: Hkv * nwork work workgroups, then Hkv * ceil(G/2) merge workgroups.  Every
// workgroup first builds the plan of its KV head in LDS (bitmaps of A and P, the
// missed list in A's order, the chunks of P that hold a wasted page).
// Work unit u < ceil(|M|/C): attend missed pages [uC, uC+C).
// Work unit u >= that (exact mode): one contaminated chunk c of P: attend its wasted
//   pages W; if they carry at most kMaxWastedShare of the chunk's softmax mass for every
//   head, subtract them from the chunk's speculative state (the clean part's maximum
//   comes from the per-page maxima of the speculation); otherwise attend the chunk's
//   pages of A afresh.  Either way the unit's state replaces chunk c.
// Merge workgroups wait (bounded spin) until every work workgroup of their KV head has
// published its state, merge the clean chunks and all unit states, and write the output.

constexpr float kMaxWastedShare = 0.875f;
constexpr int kSpinLimit = 1 << 24;

struct RepairLds {
  uint32_t bitA[PRR_MAX_PAGES_DEV / 32];
  uint32_t bitP[PRR_MAX_PAGES_DEV / 32];
  int32_t listP[PRR_MAX_CAP_DEV];
  int32_t missed[PRR_MAX_CAP_DEV];
  int32_t contam[PRR_MAX_CAP_DEV];
  uint32_t contam_bits[PRR_MAX_CAP_DEV / 32];
  uint8_t wflag[PRR_MAX_CAP_DEV];
  int cnt_m[4][4], cnt_w[4][4], cnt_c[4][4];
  int32_t wpages[16];
  int32_t xpages[16];
  int32_t xslots[16];
  float fred[2][16];
  int nWp, nXp;
  union {
    UnitLds unit;  // work workgroups
    struct {       // merge workgroups: each wave's running state
      float acc[4][kHeadDim];
      float ml[4][2];
    } merge;
  };
};

// A wave's share of a merge: the states i = par, par + 2, .. < n folded into the running
// (M, L, ax, ay), where ml(i, m, l) loads state i's (m, l) and out(i) its outputs at
// columns 2 lane and 2 lane + 1.  Each batch issues the loads of up to 32 states before
// using any of them, so it costs one memory round trip.
template <class ML, class OUT>
__device__ __forceinline__ void fold_states(int n, int par, const ML& ml, const OUT& out, float& M, float& L, float& ax,
                                            float& ay) {
  const float kNegInf = -__builtin_inff();
  const int lane = lane_id();
  const int nk = n > par ? (n - par + 1) / 2 : 0;
  for (int k0 = 0; k0 < nk; k0 += 32) {
    const int nb = min(32, nk - k0);
    float mi, li;
    ml(par + 2 * (k0 + min(lane, nb - 1)), mi, li);
    float2 ov[32];
#pragma unroll
    for (int r = 0; r < 32; ++r) ov[r] = out(par + 2 * (k0 + min(r, nb - 1)));
    li = lane < nb ? li : 0.0f;
    mi = li > 0.0f ? mi : kNegInf;
    const float Mn = fmaxf(M, wave_max(mi));
    if (Mn == kNegInf) continue;  // no state of this batch holds anything
    const float sc = L > 0.0f ? exp2f((M - Mn) * kLog2e) : 0.0f;
    const float wi = li > 0.0f ? li * exp2f((mi - Mn) * kLog2e) : 0.0f;
    ax *= sc;
    ay *= sc;
    L = L * sc + wave_sum(wi);
    M = Mn;
#pragma unroll
    for (int r = 0; r < 32; ++r) {
      const float wr = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wi), r));
      ax += wr * ov[r].x;
      ay += wr * ov[r].y;
    }
  }
}

template <bool BF16, int PS>
__global__ __launch_bounds__(256) void repair_kernel(const RepairLaunch a) {
  __shared__ RepairLds S;
  const int t = threadIdx.x, lane = lane_id(), w = t / kWave;
  const int G = a.group, C = a.chunk;
  const int work_wgs = a.num_kv_heads * a.nwork;
  const int bid = blockIdx.x;
  const bool is_merge = bid >= work_wgs;
  int h, u = 0, pair = 0;
  if (!is_merge) {
    h = bid / a.nwork;
    u = bid % a.nwork;
  } else {
    const int m = bid - work_wgs;
    h = m / a.nmerge_per_kv;
    pair = m % a.nmerge_per_kv;
  }
  const bool exact = a.mode == PRR_EXACT_SELECTED;
  const int n = a.num_pages;
  const int nwords = (n + 31) / 32;
  const int nA = min(max(a.selected_count[h], 0), a.cap);
  const int nP = a.predicted ? min(max(a.predicted_count[h], 0), a.cap) : 0;
  const float kNegInf = -__builtin_inff();

  // ---- plan.  List entry i is handled by thread i % 256 in round i / 256, so a wave
  // covers 64 consecutive entries and every compaction is a ballot.
  for (int i = t; i < nwords; i += 256) {
    S.bitA[i] = 0u;
    S.bitP[i] = 0u;
  }
  // the list entries are loaded together with the counts (clamped to the capacity) and
  // masked afterwards, so the plan costs one memory round trip
  int ea[4], ep[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const size_t ic = (size_t)h * a.cap + min(r * 256 + t, a.cap - 1);
    ea[r] = a.selected[ic];
    ep[r] = a.predicted ? a.predicted[ic] : -1;
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int i = r * 256 + t;
    ea[r] = i < nA ? ea[r] : -1;
    ep[r] = i < nP ? ep[r] : -1;
  }
  __syncthreads();
  bool bad_entry = false;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int i = r * 256 + t;
    if (i < nA) {
      if (ea[r] >= 0 && ea[r] < n) atomicOr(&S.bitA[ea[r] >> 5], 1u << (ea[r] & 31));
      else bad_entry = true;
    }
    if (i < nP) {
      S.listP[i] = ep[r];
      if (ep[r] >= 0 && ep[r] < n) atomicOr(&S.bitP[ep[r] >> 5], 1u << (ep[r] & 31));
      else bad_entry = true;
    }
  }
  if (bad_entry && bid == 0) atomicOr(a.flags, kFlagBadListEntry);
  __syncthreads();
  uint64_t bm[4], bw[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int i = r * 256 + t;
    const int pa = ea[r], pp = ep[r];
    const bool missed = i < nA && pa >= 0 && pa < n && !((S.bitP[pa >> 5] >> (pa & 31)) & 1u);
    const bool wasted = i < nP && pp >= 0 && pp < n && !((S.bitA[pp >> 5] >> (pp & 31)) & 1u);
    if (i < nP) S.wflag[i] = wasted ? 1 : 0;
    bm[r] = __ballot(missed);
    bw[r] = __ballot(wasted);
    if (lane == 0) {
      S.cnt_m[r][w] = __popcll(bm[r]);
      S.cnt_w[r][w] = __popcll(bw[r]);
    }
  }
  __syncthreads();
  int nM = 0, nW = 0;
  {
    int base[4] = {0, 0, 0, 0};
#pragma unroll
    for (int r = 0; r < 4; ++r) {
#pragma unroll
      for (int ww = 0; ww < 4; ++ww) {
        if (r < 0 || ww < 0) continue;
        const int c = S.cnt_m[r][ww];
#pragma unroll
        for (int rr = 0; rr < 4; ++rr)
          if (r < rr || (r == rr && ww < w)) base[rr] += c;
        nM += c;
        nW += S.cnt_w[r][ww];
      }
    }
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if ((bm[r] >> lane) & 1ull) S.missed[base[r] + lanes_below(bm[r])] = ea[r];
  }
  const int nch = (nP + C - 1) / C;
  int nCont = 0;
  if (exact) {
    // chunk c (of C consecutive entries of P) holds a wasted page: thread c % 256, round c / 256
    uint64_t bc[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int c = r * 256 + t;
      bool dirty = false;
      if (c < nch) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int i = c * C + e;
          if (e < C && i < nP) dirty |= S.wflag[i] != 0;
        }
      }
      bc[r] = __ballot(dirty);
      if (lane == 0) S.cnt_c[r][w] = __popcll(bc[r]);
    }
    for (int i = t; i < PRR_MAX_CAP_DEV / 32; i += 256) S.contam_bits[i] = 0u;
    __syncthreads();
    int base[4] = {0, 0, 0, 0};
#pragma unroll
    for (int r = 0; r < 4; ++r) {
#pragma unroll
      for (int ww = 0; ww < 4; ++ww) {
        const int c = S.cnt_c[r][ww];
#pragma unroll
        for (int rr = 0; rr < 4; ++rr)
          if (r < rr || (r == rr && ww < w)) base[rr] += c;
        nCont += c;
      }
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      if ((bc[r] >> lane) & 1ull) {
        const int c = r * 256 + t;
        S.contam[base[r] + lanes_below(bc[r])] = c;
        atomicOr(&S.contam_bits[c >> 5], 1u << (c & 31));
      }
    }
  }
  __syncthreads();
  const int nMU = (nM + C - 1) / C;

  AttnCtx ctx;
  ctx.q = static_cast<const uint16_t*>(a.q) + (size_t)h * G * kHeadDim;
  ctx.k = static_cast<const uint16_t*>(a.k_cache) + (size_t)h * a.max_pages * a.page_size * kHeadDim;
  ctx.v = static_cast<const uint16_t*>(a.v_cache) + (size_t)h * a.max_pages * a.page_size * kHeadDim;
  ctx.ptab = a.page_table;
  ctx.max_pages = a.max_pages;
  ctx.num_pages = n;
  ctx.num_tokens = a.num_tokens;
  ctx.G = G;
  const int hh = t >> 4, c0 = (t & 15) * 8;

  if (!is_merge) {
    // ---- work
    UnitResult r;
    bool have = false;
    if (u < nMU) {
      const int start = u * C;
      attend_unit<BF16, PS>(ctx, S.missed + start, min(C, nM - start), nullptr, S.unit, a.flags, r);
      have = true;
    } else if (exact && u - nMU < nCont) {
      const int ch = S.contam[u - nMU];
      if (t == 0) {
        int nw = 0, nx = 0;
        for (int i = ch * C; i < min(nP, ch * C + C); ++i) {
          const int p = S.listP[i];
          if (p < 0 || p >= n) continue;
          if ((S.bitA[p >> 5] >> (p & 31)) & 1u) {
            S.xpages[nx] = p;
            S.xslots[nx] = i;
            ++nx;
          } else {
            S.wpages[nw++] = p;
          }
        }
        S.nWp = nw;
        S.nXp = nx;
      }
      __syncthreads();
      const int nwp = S.nWp, nxp = S.nXp;
      bool recompute = true;
      if (a.page_m && nxp > 0 && nwp > 0) {
        // the chunk's speculative state and its kept pages' maxima are loaded before the
        // wasted pages are attended, so that their round trip overlaps the attention's
        const size_t crow = ((size_t)h * a.nchunks + ch) * G;
        float mx = kNegInf, mc = 0.f, lc = 0.f;
        float4 o0 = make_float4(0.f, 0.f, 0.f, 0.f), o1 = o0;
        if (hh < G) {
          mc = a.part_m[crow + hh];
          lc = a.part_l[crow + hh];
          const float4* oc = reinterpret_cast<const float4*>(a.part_o + (crow + hh) * kHeadDim + c0);
          o0 = oc[0];
          o1 = oc[1];
          for (int x = 0; x < nxp; ++x) mx = fmaxf(mx, a.page_m[((size_t)h * a.cap + S.xslots[x]) * G + hh]);
        }
        attend_unit<BF16, PS>(ctx, S.wpages, nwp, nullptr, S.unit, a.flags, r);
        bool bad = false;
        if (hh < G) {
          const float share = (lc > 0.f && r.l > 0.f) ? r.l * exp2f((r.m - mc) * kLog2e) / lc : (r.l > 0.f ? 2.f : 0.f);
          bad = !(share <= kMaxWastedShare);
        }
        bad = __syncthreads_or(bad);
        if (!bad) {
          recompute = false;
          if (hh < G) {
            const float ec = lc * exp2f((mc - mx) * kLog2e);
            const float ew = r.l > 0.f ? r.l * exp2f((r.m - mx) * kLog2e) : 0.f;
            const float lx = ec - ew;
            const float inv = 1.0f / lx;
            const float ocv[8] = {o0.x, o0.y, o0.z, o0.w, o1.x, o1.y, o1.z, o1.w};
#pragma unroll
            for (int e = 0; e < 8; ++e) r.o[e] = (ec * ocv[e] - ew * r.o[e]) * inv;
            r.m = mx;
            r.l = lx;
          }
        }
      }
      if (recompute) attend_unit<BF16, PS>(ctx, S.xpages, nxp, nullptr, S.unit, a.flags, r);
      have = true;
    }
    // publish the unit state to the merge workgroups: device-coherent stores, staged through
    // LDS so that each store instruction writes 256 contiguous bytes, completed before the
    // counter is bumped
    if (have) {
      float* tile = &S.unit.wo[0][0][0];  // [16][128], free after the unit's last barrier
      if (hh < G) {
#pragma unroll
        for (int e = 0; e < 8; ++e) tile[hh * kHeadDim + c0 + e] = r.o[e];
        if ((t & 15) == 0) {
          S.unit.wm[0][hh] = r.m;
          S.unit.wl[0][hh] = r.l;
        }
      }
      __syncthreads();
      float* dst = a.ws_o + ((size_t)h * a.nwork + u) * G * kHeadDim;
      for (int i = t; i < G * kHeadDim; i += 256) st_dev(dst + i, tile[i]);
      if (t < 2 * G) st_dev(a.ws_ml + (((size_t)h * a.nwork + u) * G) * 2 + t, (t & 1) ? S.unit.wl[0][t >> 1] : S.unit.wm[0][t >> 1]);
    }
    stores_complete();
    __syncthreads();
    if (t == 0) counter_add(&a.ws_cnt[h], 1u);
    return;
  }

  // ---- merge.  Wave w folds, for query head pair * 2 + (w & 1), every other state
  // (w >> 1 picks the parity): first the clean speculative chunks, which are ready at
  // launch (folded while the work workgroups run), then, once every work workgroup of the
  // KV head has published, the unit states; the two waves of a head are combined at the end.
  const int nUnits = nMU + (exact ? nCont : 0);
  const int gi = w & 1, par = w >> 1, g = pair * 2 + gi;
  const size_t crow0 = ((size_t)h * a.nchunks) * G + min(g, G - 1);
  const size_t urow0 = ((size_t)h * a.nwork) * G + min(g, G - 1);
  float Mw = kNegInf, Lw = 0.f, ax = 0.f, ay = 0.f;
  if (g < G) {
    fold_states(
        nch, par,
        [&](int c, float& m, float& l) {
          const size_t row = crow0 + (size_t)c * G;
          const bool clean = !(exact && ((S.contam_bits[c >> 5] >> (c & 31)) & 1u));
          m = a.part_m[row];
          l = clean ? a.part_l[row] : 0.0f;
        },
        [&](int c) {
          return *reinterpret_cast<const float2*>(a.part_o + (crow0 + (size_t)c * G) * kHeadDim + 2 * lane);
        },
        Mw, Lw, ax, ay);
  }
  if (t == 0) {
    int it = 0;
    while (ld_dev(&a.ws_cnt[h]) < (uint32_t)a.nwork) {
      __builtin_amdgcn_s_sleep(1);
      if (++it > kSpinLimit) {
        atomicOr(a.flags, kFlagSpinTimeout);
        break;
      }
    }
  }
  __syncthreads();
  if (g < G) {
    fold_states(
        nUnits, par,
        [&](int u, float& m, float& l) {
          const size_t row = urow0 + (size_t)u * G;
          m = ld_dev(a.ws_ml + row * 2);
          l = ld_dev(a.ws_ml + row * 2 + 1);
        },
        [&](int u) {
          const uint64_t v = __hip_atomic_load(
              reinterpret_cast<uint64_t*>(a.ws_o + (urow0 + (size_t)u * G) * kHeadDim) + lane, __ATOMIC_RELAXED,
              __HIP_MEMORY_SCOPE_AGENT);
          return make_float2(__uint_as_float((uint32_t)v), __uint_as_float((uint32_t)(v >> 32)));
        },
        Mw, Lw, ax, ay);
  }
  *reinterpret_cast<float2*>(&S.merge.acc[w][2 * lane]) = make_float2(ax, ay);
  if (lane == 0) {
    S.merge.ml[w][0] = Mw;
    S.merge.ml[w][1] = Lw;
  }
  __syncthreads();
  if (par == 0 && g < G) {
    const float m1 = S.merge.ml[w][0], l1 = S.merge.ml[w][1];
    const float m2 = S.merge.ml[w + 2][0], l2 = S.merge.ml[w + 2][1];
    const float ms = fmaxf(l1 > 0.f ? m1 : kNegInf, l2 > 0.f ? m2 : kNegInf);
    const float f1 = l1 > 0.f ? exp2f((m1 - ms) * kLog2e) : 0.f;
    const float f2 = l2 > 0.f ? exp2f((m2 - ms) * kLog2e) : 0.f;
    const float L = l1 * f1 + l2 * f2;
    const float inv = L > 0.f ? 1.0f / L : 0.f;
    const float2 o1 = *reinterpret_cast<const float2*>(&S.merge.acc[w][2 * lane]);
    const float2 o2 = *reinterpret_cast<const float2*>(&S.merge.acc[w + 2][2 * lane]);
    const float ox = (o1.x * f1 + o2.x * f2) * inv, oy = (o1.y * f1 + o2.y * f2) * inv;
    const size_t orow = (size_t)h * G + g;
    *reinterpret_cast<float2*>(a.out_o32 + orow * kHeadDim + 2 * lane) = make_float2(ox, oy);
    if (a.out_o)
      reinterpret_cast<uint32_t*>(a.out_o)[(orow * kHeadDim) / 2 + lane] = f2h_rne<BF16>(ox) | (f2h_rne<BF16>(oy) << 16);
    if (lane == 0) {
      a.out_m[orow] = L > 0.f ? ms : kNegInf;
      a.out_l[orow] = L;
    }
  }
  if (pair == 0 && t == 0) {
    if (a.missed_count) a.missed_count[h] = nM;
    if (a.wasted_count) a.wasted_count[h] = nW;
  }
  __syncthreads();
  if (t == 0) {
    const uint32_t old = atomicAdd(&a.ws_cnt[a.num_kv_heads + h], 1u);
    if (old == (uint32_t)(a.nmerge_per_kv - 1)) {
      atomicExch(&a.ws_cnt[h], 0u);
      atomicExch(&a.ws_cnt[a.num_kv_heads + h], 0u);
    }
  }
}

// =====================================================================================
// merge of arbitrary partial states
// =====================================================================================

__global__ __launch_bounds__(256) void merge_states_kernel(int n_states, int rows, int d, const float* __restrict__ o,
                                                           const float* __restrict__ m, const float* __restrict__ l,
                                                           float* __restrict__ out_o, float* __restrict__ out_m,
                                                           float* __restrict__ out_l) {
  const int row = blockIdx.x;
  const float kNegInf = -__builtin_inff();
  float ms = kNegInf;
  for (int s = 0; s < n_states; ++s) {
    const size_t i = (size_t)s * rows + row;
    if (l[i] > 0.f) ms = fmaxf(ms, m[i]);
  }
  float L = 0.f;
  for (int s = 0; s < n_states; ++s) {
    const size_t i = (size_t)s * rows + row;
    if (l[i] > 0.f) L += l[i] * exp2f((m[i] - ms) * kLog2e);
  }
  for (int c = threadIdx.x; c < d; c += blockDim.x) {
    float O = 0.f;
    for (int s = 0; s < n_states; ++s) {
      const size_t i = (size_t)s * rows + row;
      if (l[i] > 0.f) O += l[i] * exp2f((m[i] - ms) * kLog2e) * o[i * d + c];
    }
    out_o[(size_t)row * d + c] = L > 0.f ? O / L : 0.f;
  }
  if (threadIdx.x == 0) {
    out_m[row] = L > 0.f ? ms : kNegInf;
    out_l[row] = L;
  }
}

// =====================================================================================
// launchers
// =====================================================================================

// Dynamic LDS above 48 KiB needs the kernel's limit raised; the limit only ever grows,
// so after the first (eager) call of a shape no attribute call is made, which keeps
// graph capture free of them.  A failed attribute call is cleared from HIP's last-error
// state so that it is not mistaken for a launch error of the caller.
static std::mutex g_lds_mutex;
static std::map<const void*, size_t> g_lds_limit;

static void allow_lds(const void* f, size_t bytes) {
  if (bytes <= 48 * 1024) return;
  std::lock_guard<std::mutex> lock(g_lds_mutex);
  size_t& cur = g_lds_limit[f];
  if (cur >= bytes) return;
  if (hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes) == hipSuccess) cur = bytes;
  else (void)hipGetLastError();
}

// Launch a kernel taking one by-value descriptor and return the launch's own status.
template <typename A>
static hipError_t launch1(const void* f, dim3 grid, dim3 block, size_t lds, hipStream_t stream, const A& arg) {
  allow_lds(f, lds);
  void* args[] = {const_cast<A*>(&arg)};
  return hipLaunchKernel(f, grid, block, args, lds, stream);
}

hipError_t launch_score_topk(const ScoreLaunch& a, hipStream_t stream) {
  dim3 grid((a.num_pages + kScorePagesPerWg - 1) / kScorePagesPerWg, a.num_kv_heads);
  const void* f = a.bf16 ? (a.meta_mean ? (const void*)score_topk_kernel<true, true> : (const void*)score_topk_kernel<true, false>)
                         : (a.meta_mean ? (const void*)score_topk_kernel<false, true> : (const void*)score_topk_kernel<false, false>);
  return launch1(f, grid, dim3(kSelThreads), 0, stream, a);
}

hipError_t launch_predict(const PredictLaunch& a, hipStream_t stream) {
  return launch1((const void*)predict_kernel, dim3(a.num_kv_heads), dim3(kSelThreads), 0, stream, a);
}

template <bool BF16>
struct SpecK {
  template <int PS>
  static const void* get() { return (const void*)spec_attn_kernel<BF16, PS>; }
};
template <bool BF16>
struct RepairK {
  template <int PS>
  static const void* get() { return (const void*)repair_kernel<BF16, PS>; }
};

hipError_t launch_spec_attn(const SpecLaunch& a, hipStream_t stream) {
  dim3 grid(a.nchunks, a.num_kv_heads);
  const void* f = a.bf16 ? by_page_size<SpecK<true>>(a.page_size) : by_page_size<SpecK<false>>(a.page_size);
  if (!f) return hipErrorInvalidValue;
  return launch1(f, grid, dim3(256), 0, stream, a);
}

hipError_t launch_repair(const RepairLaunch& a, hipStream_t stream) {
  const int grid = a.num_kv_heads * (a.nwork + a.nmerge_per_kv);
  const void* f = a.bf16 ? by_page_size<RepairK<true>>(a.page_size) : by_page_size<RepairK<false>>(a.page_size);
  if (!f) return hipErrorInvalidValue;
  return launch1(f, dim3(grid), dim3(256), 0, stream, a);
}

hipError_t launch_merge_states(int n_states, int rows, int d, const float* o, const float* m, const float* l,
                               float* out_o, float* out_m, float* out_l, hipStream_t stream) {
  void* args[] = {&n_states, &rows, &d, &o, &m, &l, &out_o, &out_m, &out_l};
  return hipLaunchKernel((const void*)merge_states_kernel, dim3(rows), dim3(256), args, 0, stream);
}

}  // namespace prr
