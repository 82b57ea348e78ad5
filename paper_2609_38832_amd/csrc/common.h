// Shared device helpers for the gfx950 kernels: bf16 conversion, wave-level
// primitives, launch plumbing.  Internal to libnamoh.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#define NAMOH_DEV __device__ __forceinline__

namespace namoh {

constexpr int kWave = 64;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
constexpr bf16x2 kOnes2 = {static_cast<__bf16>(1.0f), static_cast<__bf16>(1.0f)};

// bf16 stored as raw 16-bit patterns in memory.
NAMOH_DEV float bf16_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// Round to nearest even; inputs here are finite.
NAMOH_DEV uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

// Two floats -> packed bf16 pair (lo in the low half).
NAMOH_DEV uint32_t pack_bf16x2(float lo, float hi) {
  return static_cast<uint32_t>(f32_to_bf16(lo)) |
         (static_cast<uint32_t>(f32_to_bf16(hi)) << 16);
}

NAMOH_DEV float lo_bf16(uint32_t w) { return __uint_as_float(w << 16); }
NAMOH_DEV float hi_bf16(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Thread / workgroup index in x, read straight from the hardware registers
// (the threadIdx / blockIdx accessors can be left as out-of-line library
// calls, which clobber registers at kernel entry).
NAMOH_DEV int thread_x() { return static_cast<int>(__builtin_amdgcn_workitem_id_x()); }
NAMOH_DEV int block_x() { return static_cast<int>(__builtin_amdgcn_workgroup_id_x()); }

// Lanes below the calling lane in a 64-wide wave.
NAMOH_DEV uint64_t lanemask_lt() {
  const int lane = __lane_id();
  return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

NAMOH_DEV int ceil_div(int a, int b) { return (a + b - 1) / b; }

// (cos, sin) of a RoPE angle given in double, in double arithmetic without
// library calls: Cody-Waite reduction by pi/2 (two-part constant, fused
// multiply-adds) to |r| <= pi/4, Taylor polynomials of degree 11 (sin) and
// 12 (cos) there (truncation below 1e-11), and the quadrant's sign/swap.
// Accurate to the final float rounding for angles below 2^30.
NAMOH_DEV float2 rope_cos_sin(double angle) {
  constexpr double kTwoOverPi = 0.6366197723675814;
  constexpr double kPiHalfHi = 1.5707963267948966;
  constexpr double kPiHalfLo = 6.123233995736766e-17;
  const double n = rint(angle * kTwoOverPi);
  double r = fma(-n, kPiHalfHi, angle);
  r = fma(-n, kPiHalfLo, r);
  const double r2 = r * r;
  const double sn =
      r * (1.0 + r2 * (-1.0 / 6 + r2 * (1.0 / 120 + r2 * (-1.0 / 5040 +
           r2 * (1.0 / 362880 + r2 * (-1.0 / 39916800))))));
  const double cs =
      1.0 + r2 * (-1.0 / 2 + r2 * (1.0 / 24 + r2 * (-1.0 / 720 + r2 * (1.0 / 40320 +
            r2 * (-1.0 / 3628800 + r2 * (1.0 / 479001600))))));
  const int q = static_cast<int>(static_cast<long long>(n) & 3);
  const double c = q == 0 ? cs : (q == 1 ? -sn : (q == 2 ? -cs : sn));
  const double s = q == 0 ? sn : (q == 1 ? cs : (q == 2 ? -sn : -cs));
  return make_float2(static_cast<float>(c), static_cast<float>(s));
}

// ---- cross-lane operations on the VALU ------------------------------------
// __shfl_* go through the LDS crossbar (ds_bpermute, one LDS round trip per
// step); these use DPP lane patterns (GFX9 controls) and the gfx950 row-swap
// instructions instead.  Patterns: quad_perm [1,0,3,2] = lane ^ 1,
// [2,3,0,1] = lane ^ 2; row_half_mirror = lane 7 - i within each 8 lanes;
// row_mirror = lane 15 - i within each row of 16; row_shr n; row_bcast15 /
// row_bcast31 (lane 15 of a row to the next row / lane 31 to rows 2 and 3);
// v_permlane16_swap / v_permlane32_swap hand every lane its own value and
// that of lane ^ 16 / lane ^ 32.
constexpr int kDppXor1 = 0xB1, kDppXor2 = 0x4E, kDppRowHalfMirror = 0x141, kDppRowMirror = 0x140;
constexpr int kDppRowShr1 = 0x111, kDppRowBcast15 = 0x142, kDppRowBcast31 = 0x143;

template <int CTRL>
NAMOH_DEV int dpp_i(int x) {
  return __builtin_amdgcn_mov_dpp(x, CTRL, 0xF, 0xF, true);
}
template <int CTRL>
NAMOH_DEV float dpp_f(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), CTRL, 0xF, 0xF, true));
}
// x from the source lane of the pattern, 0 where the source lies outside the
// row or the row is not in ROWS
template <int CTRL, int ROWS = 0xF>
NAMOH_DEV int dpp_i0(int x) {
  return __builtin_amdgcn_update_dpp(0, x, CTRL, ROWS, 0xF, false);
}

// Sum / max over aligned groups of N lanes (N = 2 .. 64), the result in every
// lane of the group; every lane forms the same operands, so the result is
// the same bit pattern in all of them.
template <int N>
NAMOH_DEV float group_sum(float x) {
  static_assert(N >= 2 && N <= 64 && (N & (N - 1)) == 0, "group size");
  x += dpp_f<kDppXor1>(x);
  if constexpr (N >= 4) x += dpp_f<kDppXor2>(x);
  if constexpr (N >= 8) x += dpp_f<kDppRowHalfMirror>(x);
  if constexpr (N >= 16) x += dpp_f<kDppRowMirror>(x);
  if constexpr (N >= 32) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  }
  if constexpr (N >= 64) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  }
  return x;
}
template <int N>
NAMOH_DEV float group_max(float x) {
  static_assert(N >= 2 && N <= 64 && (N & (N - 1)) == 0, "group size");
  x = fmaxf(x, dpp_f<kDppXor1>(x));
  if constexpr (N >= 4) x = fmaxf(x, dpp_f<kDppXor2>(x));
  if constexpr (N >= 8) x = fmaxf(x, dpp_f<kDppRowHalfMirror>(x));
  if constexpr (N >= 16) x = fmaxf(x, dpp_f<kDppRowMirror>(x));
  if constexpr (N >= 32) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
  }
  if constexpr (N >= 64) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
  }
  return x;
}
template <int N>
NAMOH_DEV int group_sum_i(int x) {
  static_assert(N >= 2 && N <= 16 && (N & (N - 1)) == 0, "group size");
  x += dpp_i<kDppXor1>(x);
  if constexpr (N >= 4) x += dpp_i<kDppXor2>(x);
  if constexpr (N >= 8) x += dpp_i<kDppRowHalfMirror>(x);
  if constexpr (N >= 16) x += dpp_i<kDppRowMirror>(x);
  return x;
}
// Sum over the 64 lanes of a wave in double (exact for integer values whose
// partial sums stay below 2^53).
template <int CTRL>
NAMOH_DEV double dpp_d(double x) {
  const unsigned long long b = static_cast<unsigned long long>(__double_as_longlong(x));
  const int lo = __builtin_amdgcn_mov_dpp(static_cast<int>(static_cast<uint32_t>(b)), CTRL, 0xF, 0xF, true);
  const int hi = __builtin_amdgcn_mov_dpp(static_cast<int>(static_cast<uint32_t>(b >> 32)), CTRL, 0xF, 0xF, true);
  return __longlong_as_double(static_cast<long long>(
      (static_cast<unsigned long long>(static_cast<uint32_t>(hi)) << 32) | static_cast<uint32_t>(lo)));
}
NAMOH_DEV double wave_sum_d(double x) {
  x += dpp_d<kDppXor1>(x);
  x += dpp_d<kDppXor2>(x);
  x += dpp_d<kDppRowHalfMirror>(x);
  x += dpp_d<kDppRowMirror>(x);
  const unsigned long long b = static_cast<unsigned long long>(__double_as_longlong(x));
  const uint32_t lo = static_cast<uint32_t>(b), hi = static_cast<uint32_t>(b >> 32);
  const auto l16 = __builtin_amdgcn_permlane16_swap(lo, lo, false, false);
  const auto h16 = __builtin_amdgcn_permlane16_swap(hi, hi, false, false);
  auto mk = [](uint32_t l, uint32_t h) {
    return __longlong_as_double(static_cast<long long>((static_cast<unsigned long long>(h) << 32) | l));
  };
  x = mk(l16[0], h16[0]) + mk(l16[1], h16[1]);
  const unsigned long long c = static_cast<unsigned long long>(__double_as_longlong(x));
  const uint32_t lo2 = static_cast<uint32_t>(c), hi2 = static_cast<uint32_t>(c >> 32);
  const auto l32 = __builtin_amdgcn_permlane32_swap(lo2, lo2, false, false);
  const auto h32 = __builtin_amdgcn_permlane32_swap(hi2, hi2, false, false);
  return mk(l32[0], h32[0]) + mk(l32[1], h32[1]);
}
NAMOH_DEV int wave_max_i(int x) {
  x = max(x, dpp_i<kDppXor1>(x));
  x = max(x, dpp_i<kDppXor2>(x));
  x = max(x, dpp_i<kDppRowHalfMirror>(x));
  x = max(x, dpp_i<kDppRowMirror>(x));
  auto r = __builtin_amdgcn_permlane16_swap(static_cast<uint32_t>(x), static_cast<uint32_t>(x), false, false);
  x = max(static_cast<int>(r[0]), static_cast<int>(r[1]));
  r = __builtin_amdgcn_permlane32_swap(static_cast<uint32_t>(x), static_cast<uint32_t>(x), false, false);
  return max(static_cast<int>(r[0]), static_cast<int>(r[1]));
}

// Inclusive scan across a 64-lane wave: Kogge-Stone inside each row of 16
// (row_shr 1, 2, 4, 8), then row 0's total into row 1 and row 2's into row 3
// (row_bcast15), then the first 32 lanes' total into rows 2 and 3
// (row_bcast31).
NAMOH_DEV int wave_inclusive_scan(int x) {
  x += dpp_i0<kDppRowShr1>(x);
  x += dpp_i0<kDppRowShr1 + 1>(x);
  x += dpp_i0<kDppRowShr1 + 3>(x);
  x += dpp_i0<kDppRowShr1 + 7>(x);
  x += dpp_i0<kDppRowBcast15, 0xA>(x);
  x += dpp_i0<kDppRowBcast31, 0xC>(x);
  return x;
}

// Exclusive scan of one int per thread across a workgroup of NT threads.
// `s_wave` must hold NT/64 ints; returns the exclusive prefix and sets
// `total`.  Contains barriers: every thread of the block must call it.
template <int NT>
NAMOH_DEV int block_exclusive_scan(int x, int* s_wave, int& total) {
  static_assert(NT % kWave == 0 && NT / kWave <= kWave, "block size");
  const int lane = __lane_id();
  const int wave = thread_x() / kWave;
  const int incl = wave_inclusive_scan(x);
  if (lane == kWave - 1) s_wave[wave] = incl;
  __syncthreads();
  if (wave == 0) {
    const int wv = lane < NT / kWave ? s_wave[lane] : 0;
    const int wi = wave_inclusive_scan(wv);
    if (lane < NT / kWave) s_wave[lane] = wi - wv;
    if (lane == NT / kWave - 1) s_wave[NT / kWave] = wi;  // block total
  }
  __syncthreads();
  const int r = s_wave[wave] + incl - x;
  total = s_wave[NT / kWave];
  __syncthreads();
  return r;
}

}  // namespace namoh
