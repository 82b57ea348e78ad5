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

// Inclusive scan across a 64-lane wave.
NAMOH_DEV int wave_inclusive_scan(int x) {
  const int lane = __lane_id();
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const int y = __shfl_up(x, o, kWave);
    if (lane >= o) x += y;
  }
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
