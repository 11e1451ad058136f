// device_util.hpp -- small gfx950 device helpers shared by the SparDA kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sparda {

constexpr int kWave = 64;        // CDNA wavefront width
constexpr int kHeadDim = 128;    // D
constexpr int kBlock = 64;       // tokens per KV block

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// ---- bf16 <-> float -------------------------------------------------------------------

__device__ __forceinline__ float bf16lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// float -> bf16, round to nearest even (finite inputs; NaN stays NaN).
__device__ __forceinline__ uint16_t f32_to_bf16(float x) {
  uint32_t u = __float_as_uint(x);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// float64 -> bf16 in one rounding (nearest, ties to even), by integer work on the float64 bits,
// so that an exact float64 value is never rounded twice.
__device__ __forceinline__ uint16_t f64_to_bf16(double x) {
  const uint64_t u = (uint64_t)__double_as_longlong(x);
  const uint16_t sign = (uint16_t)((u >> 48) & 0x8000u);
  const int e = (int)((u >> 52) & 0x7ff);
  const uint64_t man = u & ((1ull << 52) - 1);
  if (e == 0x7ff) return (uint16_t)(sign | (man ? 0x7fc0u : 0x7f80u));
  if (e == 0) return sign;  // float64 subnormals are far below the bf16 range
  int be = e - 1023 + 127;
  if (be >= 1) {
    uint64_t keep = man >> 45;
    const uint64_t rest = man & ((1ull << 45) - 1), half = 1ull << 44;
    if (rest > half || (rest == half && (keep & 1u))) ++keep;
    if (keep == 128) { keep = 0; ++be; }
    if (be >= 255) return (uint16_t)(sign | 0x7f80u);
    return (uint16_t)(sign | (uint16_t)(be << 7) | (uint16_t)keep);
  }
  // bf16 subnormal: value = sig * 2^(e - 1075), grid 2^-133 => q = sig >> (942 - e), rounded.
  const uint64_t sig = man | (1ull << 52);
  const int sh = 942 - e;  // >= 46 here
  if (sh >= 64) return sign;
  uint64_t q = sig >> sh;
  const uint64_t rest = sig & ((1ull << sh) - 1), half = 1ull << (sh - 1);
  if (rest > half || (rest == half && (q & 1u))) ++q;
  return (uint16_t)(sign | (uint16_t)q);
}

// Order-preserving map of a float score to uint32 (larger score -> larger key); -0 maps like +0.
__device__ __forceinline__ uint32_t score_key(float s) {
  uint32_t u = __float_as_uint(s == 0.0f ? 0.0f : s);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// ---- cross-lane helpers ----------------------------------------------------------------

// DPP move within 16-lane rows (row_ror:n has control 0x120 + n).
template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), CTRL, 0xf, 0xf, false));
}

// Sum over each 16-lane row; every lane of the row receives the row total.
__device__ __forceinline__ float row16_sum(float x) {
  x += dpp_f<0x128>(x);  // row_ror:8
  x += dpp_f<0x124>(x);  // row_ror:4
  x += dpp_f<0x122>(x);  // row_ror:2
  x += dpp_f<0x121>(x);  // row_ror:1
  return x;
}

template <int CTRL>
__device__ __forceinline__ int dpp_i(int x) {
  return __builtin_amdgcn_mov_dpp(x, CTRL, 0xf, 0xf, false);
}

// Reductions over aligned groups of 8 lanes (every lane of the group receives the result):
// quad_perm [1,0,3,2], quad_perm [2,3,0,1], then row_half_mirror (lane i <-> 7-i of the group).
__device__ __forceinline__ float group8_sum(float x) {
  x += dpp_f<0xB1>(x);
  x += dpp_f<0x4E>(x);
  x += dpp_f<0x141>(x);
  return x;
}
__device__ __forceinline__ int group8_sum(int x) {
  x += dpp_i<0xB1>(x);
  x += dpp_i<0x4E>(x);
  x += dpp_i<0x141>(x);
  return x;
}

__device__ __forceinline__ int row16_sum(int x) {
  x += dpp_i<0x128>(x);  // row_ror:8
  x += dpp_i<0x124>(x);  // row_ror:4
  x += dpp_i<0x122>(x);  // row_ror:2
  x += dpp_i<0x121>(x);  // row_ror:1
  return x;
}

__device__ __forceinline__ uint32_t row16_max(uint32_t x) {
  x = max(x, (uint32_t)dpp_i<0x128>((int)x));  // row_ror:8
  x = max(x, (uint32_t)dpp_i<0x124>((int)x));  // row_ror:4
  x = max(x, (uint32_t)dpp_i<0x122>((int)x));  // row_ror:2
  x = max(x, (uint32_t)dpp_i<0x121>((int)x));  // row_ror:1
  return x;
}

__device__ __forceinline__ uint32_t row16_min(uint32_t x) {
  x = min(x, (uint32_t)dpp_i<0x128>((int)x));  // row_ror:8
  x = min(x, (uint32_t)dpp_i<0x124>((int)x));  // row_ror:4
  x = min(x, (uint32_t)dpp_i<0x122>((int)x));  // row_ror:2
  x = min(x, (uint32_t)dpp_i<0x121>((int)x));  // row_ror:1
  return x;
}

// Inclusive prefix sum over the wavefront on DPP: row_shr 1, 2, 4, 8 inside each 16-lane row
// (lanes shifted in from outside the row add 0), then row_bcast:15 adds row r's last lane to row
// r + 1 (rows 1 and 3), and row_bcast:31 adds lane 31 to rows 2 and 3.
__device__ __forceinline__ int wave_incl_scan_dpp(int x) {
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, true);  // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, true);  // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, true);  // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, true);  // row_shr:8
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false);  // row_bcast:15, rows 1 and 3
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false);  // row_bcast:31, rows 2 and 3
  return x;
}

// Exclusive prefix sum within each 16-lane row; sub = lane index inside the row.
__device__ __forceinline__ int row16_excl_scan(int x, int sub) {
  int incl = x;
  int y = __builtin_amdgcn_update_dpp(0, incl, 0x111, 0xf, 0xf, true);  // row_shr:1
  if (sub >= 1) incl += y;
  y = __builtin_amdgcn_update_dpp(0, incl, 0x112, 0xf, 0xf, true);      // row_shr:2
  if (sub >= 2) incl += y;
  y = __builtin_amdgcn_update_dpp(0, incl, 0x114, 0xf, 0xf, true);      // row_shr:4
  if (sub >= 4) incl += y;
  y = __builtin_amdgcn_update_dpp(0, incl, 0x118, 0xf, 0xf, true);      // row_shr:8
  if (sub >= 8) incl += y;
  return incl - x;
}

// Exclusive prefix sum within aligned 8-lane groups; sub = lane index inside the group.
__device__ __forceinline__ int group8_excl_scan(int x, int sub) {
  int incl = x;
  int y = __builtin_amdgcn_update_dpp(0, incl, 0x111, 0xf, 0xf, true);  // row_shr:1
  if (sub >= 1) incl += y;
  y = __builtin_amdgcn_update_dpp(0, incl, 0x112, 0xf, 0xf, true);      // row_shr:2
  if (sub >= 2) incl += y;
  y = __builtin_amdgcn_update_dpp(0, incl, 0x114, 0xf, 0xf, true);      // row_shr:4
  if (sub >= 4) incl += y;
  return incl - x;
}

// Inverse of score_key.
__device__ __forceinline__ float key_value(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

__device__ __forceinline__ int wave_incl_scan(int x) {
  const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    const int y = __shfl_up(x, d, kWave);
    if (lane >= d) x += y;
  }
  return x;
}

// Number of set bits of `mask` below this lane.
__device__ __forceinline__ int mbcnt64(uint64_t mask) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

__device__ __forceinline__ int readlane_i(int x, int lane) { return __builtin_amdgcn_readlane(x, lane); }
__device__ __forceinline__ float readlane_f(float x, int lane) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), lane));
}

// Order this wave's LDS accesses: wait for outstanding LDS operations, then a wave barrier.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0), other counters untouched
  __builtin_amdgcn_wave_barrier();
  __asm__ __volatile__("" ::: "memory");
}

__device__ __forceinline__ uint4 ld16(const void* p) { return *reinterpret_cast<const uint4*>(p); }

// The same load with the non-temporal hint, for bytes a launch reads exactly once (the decode
// K/V blocks and compressed keys): streamed data then displaces less of what the caches hold
// (measured on the 128K decode layer: attention 98.7 -> 93.0 us).
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ld16_nt(const void* p) {
  const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
  return make_uint4(v[0], v[1], v[2], v[3]);
}

// z with P(Z > z) = p for a standard normal Z (rational approximation of Abramowitz and Stegun
// 26.2.23, |error| < 4.5e-4).  Only a first guess for the exact searches that use it.
__device__ __forceinline__ float upper_normal_quantile(float p) {
  p = fminf(fmaxf(p, 1e-7f), 1.f - 1e-7f);
  const bool upper = p <= 0.5f;
  const float q = upper ? p : 1.f - p;
  const float t = __builtin_amdgcn_sqrtf(-1.3862944f * __builtin_amdgcn_logf(q));  // -2 ln q
  const float z = t - (2.515517f + t * (0.802853f + t * 0.010328f)) /
                          (1.f + t * (1.432788f + t * (0.189269f + t * 0.001308f)));
  return upper ? z : -z;
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 w) { return __builtin_bit_cast(bf16x8, w); }

__device__ __forceinline__ f32x4 mfma16x16x32(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

}  // namespace sparda
