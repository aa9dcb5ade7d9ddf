// Device-side helpers shared by the gfx950 kernels: 16-bit storage conversions,
// order-preserving score keys, wave64 reductions and scans, block scans.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace prr {

constexpr int kHeadDim = 128;
constexpr int kWave = 64;
constexpr float kLog2e = 1.4426950408889634f;

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(8))) _Float16 f16x8_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4_t;
typedef __attribute__((ext_vector_type(4))) short s16x4_t;

// ------------------------------------------------------------------ 16-bit storage

template <bool BF16>
__device__ __forceinline__ float h2f(uint32_t bits16) {
  if constexpr (BF16) {
    return __uint_as_float(bits16 << 16);
  } else {
    return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(bits16)));
  }
}

// Exact conversion back to storage for values that came from storage (min / max).
template <bool BF16>
__device__ __forceinline__ uint32_t f2h_exact(float f) {
  if constexpr (BF16) {
    return __float_as_uint(f) >> 16;
  } else {
    return __builtin_bit_cast(uint16_t, static_cast<_Float16>(f));
  }
}

// Round-to-nearest-even conversion of an arbitrary float to storage.
template <bool BF16>
__device__ __forceinline__ uint32_t f2h_rne(float f) {
  if constexpr (BF16) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;  // quiet NaN
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
  } else {
    return __builtin_bit_cast(uint16_t, static_cast<_Float16>(f));
  }
}

// Element e (0..7) of eight 16-bit values packed in a uint4.
template <bool BF16>
__device__ __forceinline__ float u4_elem(const uint4& v, int e) {
  const uint32_t w = (e < 2) ? v.x : (e < 4) ? v.y : (e < 6) ? v.z : v.w;
  return h2f<BF16>((e & 1) ? (w >> 16) : (w & 0xffffu));
}

// ------------------------------------------------------------------ score keys

// Order-preserving map of a float to uint32 (larger float -> larger key); -0 and +0
// map to the same key, so equal scores tie and fall back to the page index.
__device__ __forceinline__ uint32_t score_key(float f) {
  if (f == 0.0f) f = 0.0f;
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// ------------------------------------------------------------------ wave64 helpers

__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

__device__ __forceinline__ int lanes_below(uint64_t mask) {
  const int lane = lane_id();
  return __popcll(mask & ((1ull << lane) - 1ull));
}

// Cross-lane data movement without the LDS crossbar: DPP within 16-lane rows and the
// gfx950 permlane swaps across rows.  Every combine pairs commutative operands, so all
// participating lanes end with bitwise identical results.
constexpr int kDppXor1 = 0xB1;        // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;        // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141; // lane i <-> 7-i within each half row
constexpr int kDppMirror = 0x140;     // lane i <-> 15-i within each row
constexpr int kDppShr1 = 0x111, kDppShr2 = 0x112, kDppShr4 = 0x114, kDppShr8 = 0x118;
constexpr int kDppBcast15 = 0x142, kDppBcast31 = 0x143;

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xf, 0xf, false);
}
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xf, 0xf, false));
}

// combine over the 16 lanes of a row (all 16 lanes get the result)
__device__ __forceinline__ float sum16(float v) {
  v += dpp_f32<kDppXor1>(v);
  v += dpp_f32<kDppXor2>(v);
  v += dpp_f32<kDppHalfMirror>(v);
  v += dpp_f32<kDppMirror>(v);
  return v;
}
__device__ __forceinline__ float max16(float v) {
  v = fmaxf(v, dpp_f32<kDppXor1>(v));
  v = fmaxf(v, dpp_f32<kDppXor2>(v));
  v = fmaxf(v, dpp_f32<kDppHalfMirror>(v));
  v = fmaxf(v, dpp_f32<kDppMirror>(v));
  return v;
}
__device__ __forceinline__ float min16(float v) {
  v = fminf(v, dpp_f32<kDppXor1>(v));
  v = fminf(v, dpp_f32<kDppXor2>(v));
  v = fminf(v, dpp_f32<kDppHalfMirror>(v));
  v = fminf(v, dpp_f32<kDppMirror>(v));
  return v;
}

// combine of lanes l, l^16, l^32, l^48 (the four rows), result in all of them
__device__ __forceinline__ float sum_rows(float v) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}
__device__ __forceinline__ float max_rows(float v) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float min_rows(float v) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fminf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fminf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ uint32_t umin_rows(uint32_t v) {
  const auto a = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  v = min((uint32_t)a[0], (uint32_t)a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return min((uint32_t)b[0], (uint32_t)b[1]);
}
__device__ __forceinline__ uint32_t umax_rows(uint32_t v) {
  const auto a = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  v = max((uint32_t)a[0], (uint32_t)a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return max((uint32_t)b[0], (uint32_t)b[1]);
}
__device__ __forceinline__ int isum_rows(int v) {
  const auto a = __builtin_amdgcn_permlane16_swap((uint32_t)v, (uint32_t)v, false, false);
  v = (int)a[0] + (int)a[1];
  const auto b = __builtin_amdgcn_permlane32_swap((uint32_t)v, (uint32_t)v, false, false);
  return (int)b[0] + (int)b[1];
}

// whole-wave reductions, result in every lane
__device__ __forceinline__ float wave_sum(float v) { return sum_rows(sum16(v)); }
__device__ __forceinline__ float wave_max(float v) { return max_rows(max16(v)); }
__device__ __forceinline__ uint32_t wave_umin(uint32_t v) {
  v = min(v, dpp_u32<kDppXor1>(v));
  v = min(v, dpp_u32<kDppXor2>(v));
  v = min(v, dpp_u32<kDppHalfMirror>(v));
  v = min(v, dpp_u32<kDppMirror>(v));
  return umin_rows(v);
}
__device__ __forceinline__ uint32_t wave_umax(uint32_t v) {
  v = max(v, dpp_u32<kDppXor1>(v));
  v = max(v, dpp_u32<kDppXor2>(v));
  v = max(v, dpp_u32<kDppHalfMirror>(v));
  v = max(v, dpp_u32<kDppMirror>(v));
  return umax_rows(v);
}
__device__ __forceinline__ int wave_isum(int v) {
  v += (int)dpp_u32<kDppXor1>((uint32_t)v);
  v += (int)dpp_u32<kDppXor2>((uint32_t)v);
  v += (int)dpp_u32<kDppHalfMirror>((uint32_t)v);
  v += (int)dpp_u32<kDppMirror>((uint32_t)v);
  return isum_rows(v);
}

// inclusive prefix sum over the wave (row shifts, then the row broadcasts)
__device__ __forceinline__ int wave_inclusive_scan(int x) {
  x += (int)dpp_u32<kDppShr1>((uint32_t)x);
  x += (int)dpp_u32<kDppShr2>((uint32_t)x);
  x += (int)dpp_u32<kDppShr4>((uint32_t)x);
  x += (int)dpp_u32<kDppShr8>((uint32_t)x);
  x += __builtin_amdgcn_update_dpp(0, x, kDppBcast15, 0xa, 0xf, false);
  x += __builtin_amdgcn_update_dpp(0, x, kDppBcast31, 0xc, 0xf, false);
  return x;
}

// Block-wide exclusive scan of one int per thread; `wave_tot` needs NT/64 ints of LDS.
// Returns the exclusive prefix; `total` receives the sum over the block.
template <int NT>
__device__ __forceinline__ int block_exclusive_scan(int v, int* wave_tot, int& total) {
  constexpr int NW = NT / kWave;
  const int w = threadIdx.x / kWave;
  const int inc = wave_inclusive_scan(v);
  if (lane_id() == kWave - 1) wave_tot[w] = inc;
  __syncthreads();
  int base = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    const int s = wave_tot[i];
    base += (i < w) ? s : 0;
    tot += s;
  }
  __syncthreads();
  total = tot;
  return base + inc - v;
}

template <int NT>
__device__ __forceinline__ int block_sum(int v, int* wave_tot) {
  int total;
  block_exclusive_scan<NT>(v, wave_tot, total);
  return total;
}

template <int NT>
__device__ __forceinline__ void block_minmax_u32(uint32_t& lo, uint32_t& hi, uint32_t* scratch) {
  constexpr int NW = NT / kWave;
  lo = wave_umin(lo);
  hi = wave_umax(hi);
  const int w = threadIdx.x / kWave;
  if (lane_id() == 0) {
    scratch[w] = lo;
    scratch[NW + w] = hi;
  }
  __syncthreads();
  lo = 0xffffffffu;
  hi = 0u;
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    lo = min(lo, scratch[i]);
    hi = max(hi, scratch[NW + i]);
  }
  __syncthreads();
}

// ------------------------------------------------------------------ cross-workgroup publishing
// Data that one workgroup hands to another inside the same launch is written with
// device-coherent stores (they bypass the per-XCD L2s' non-coherent caching), the
// writer waits for its stores to complete before it bumps a counter, and the reader
// loads the data with device-coherent loads after it has observed the counter.  This
// avoids the whole-L2 write-back and invalidate of a device-scope fence.

__device__ __forceinline__ void st_dev(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_dev(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t ld_dev(const uint32_t* p) {
  return __hip_atomic_load(const_cast<uint32_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// every store of this thread has completed before anything after this point is issued
__device__ __forceinline__ void stores_complete() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0);
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}
__device__ __forceinline__ uint32_t counter_add(uint32_t* p, uint32_t v) {
  return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Sticky error bits written by kernels into the workspace flag word.
constexpr uint32_t kFlagBadListEntry = 1u;
constexpr uint32_t kFlagSpinTimeout = 2u;

// ------------------------------------------------------------------ P.V of one tile
// O^T (128 channels x 16 heads) += V^T . P^T over a tile of 16 tokens.  Lane 16j+m holds
// V rows 4j..4j+3 (channels 8m..8m+7, one 16-byte load per row) in v[0..3], and the softmax
// weights of head m for tokens 4j..4j+3 in p[0..3]; accumulator cb, register i then holds
// O[head m][32j + 8i + cb] (each lane owns the channels of the head whose weights it holds).
//
// One 16x16x16 MFMA in the cache's 16-bit type per accumulator and weight term: its A
// operand, channel 8m + cb of the lane's four rows, needs no data from other lanes, and
// the weights (in [0, 1]) are split into two terms of that type, hi = rne(p) and
// lo = rne(p - hi).  bfloat16 terms carry p to about 2^-17 relative; float16 terms to
// 2^-22 relative or 2^-25 absolute (lo is subnormal below 2^-14), far inside the
// tolerance of the outputs.  Two MFMAs replace the four fp32 16x16x4 MFMAs that a float32
// weight operand needs, at an eighth of their issue cycles.
template <bool BF16>
__device__ __forceinline__ void pv_tile(f32x4_t (&acc)[8], const u32x4_t (&v)[4], const float (&p)[4]) {
  uint32_t hi[4], lo[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    hi[i] = f2h_rne<BF16>(p[i]);
    lo[i] = f2h_rne<BF16>(p[i] - h2f<BF16>(hi[i]));
  }
  const s16x4_t bh =
      __builtin_bit_cast(s16x4_t, (uint64_t)(hi[0] | (hi[1] << 16)) | ((uint64_t)(hi[2] | (hi[3] << 16)) << 32));
  const s16x4_t bl =
      __builtin_bit_cast(s16x4_t, (uint64_t)(lo[0] | (lo[1] << 16)) | ((uint64_t)(lo[2] | (lo[3] << 16)) << 32));
#pragma unroll
  for (int cb = 0; cb < 8; ++cb) {
    const int w = cb >> 1, sh = (cb & 1) * 16;
    const uint32_t a0 = ((v[0][w] >> sh) & 0xffffu) | (((v[1][w] >> sh) & 0xffffu) << 16);
    const uint32_t a1 = ((v[2][w] >> sh) & 0xffffu) | (((v[3][w] >> sh) & 0xffffu) << 16);
    const s16x4_t va = __builtin_bit_cast(s16x4_t, (uint64_t)a0 | ((uint64_t)a1 << 32));
    if constexpr (BF16) {
      acc[cb] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(va, bh, acc[cb], 0, 0, 0);
      acc[cb] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(va, bl, acc[cb], 0, 0, 0);
    } else {
      typedef __attribute__((ext_vector_type(4))) _Float16 f16x4_t;
      acc[cb] = __builtin_amdgcn_mfma_f32_16x16x16f16(__builtin_bit_cast(f16x4_t, va), __builtin_bit_cast(f16x4_t, bh),
                                                      acc[cb], 0, 0, 0);
      acc[cb] = __builtin_amdgcn_mfma_f32_16x16x16f16(__builtin_bit_cast(f16x4_t, va), __builtin_bit_cast(f16x4_t, bl),
                                                      acc[cb], 0, 0, 0);
    }
  }
}

}  // namespace prr
