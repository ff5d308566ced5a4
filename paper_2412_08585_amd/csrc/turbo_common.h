// Device-side building blocks of the gfx950 TurboAttention kernels.
//
// Nothing here is shared with the CPU oracle; the paper's constants are typed
// again below as exact binary32 literals.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "turbo_attn.h"

namespace turbo {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef unsigned short u16;
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4_t __attribute__((ext_vector_type(4)));

// ceil(a / b) for a >= 0, b > 0, without overflow near INT_MAX.
__host__ __device__ constexpr int ceil_div(int a, int b) { return a / b + (a % b != 0); }

// Symmetric int8 divisor of Algorithms 1 and 2.
constexpr float kQmax = 119.0f;
// 1.5 * 2^23: adding it to a value of magnitude < 2^22 leaves the value
// rounded to an integer (ties to even) in the low mantissa bits.
constexpr float kMagic = 12582912.0f;
constexpr int kMagicBits = 0x4B400000;

// Accumulator seed of the i8 MFMAs: the bits of binary32 1/(2 pi) =
// 0x1.45f306p-3, one of the instruction set's inline constants.  An int32
// result seed + s with -2292099 <= s <= 6096508 stays in the binade of the
// seed (whose mantissa field is 2292099), so read as a float it is
// 0x1.45f306p-3 + s * 2^-26, and subtracting the seed gives s * 2^-26
// exactly: a full-rate subtraction replaces the half-rate int -> float
// conversion.  Every product sum here is within |s| <= 128 * 128 * 128 = 2^21.
constexpr int kAccSeed = 0x3E22F983;
constexpr float kAccSeedF = 0x1.45f306p-3f;

// s * 2^-26 of a seeded accumulator entry (exact).
__device__ __forceinline__ float acc_unseed(int r) { return __int_as_float(r) - kAccSeedF; }

// -s * 2^-26 (exact): the seed minus the entry, which takes the seed as the
// inline constant 1/(2 pi) (the subtraction the other way round needs a
// 32-bit literal).  Callers multiply by the negated factor.
__device__ __forceinline__ float acc_unseed_neg(int r) { return kAccSeedF - __int_as_float(r); }

// Ordering of one wave's own LDS exchanges (lanes writing what other lanes
// of the same wave read next): the LDS executes a wave's accesses in order,
// so only the compiler has to be kept from reordering them -- no s_barrier
// and no wait, unlike __syncthreads.
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// SAS (Sec. 4): e^{-y} ~ LUT[floor y] * POLY(y - floor y) for y = m - s in
// [0, 6]; zero for y > 6 (n_r = -6, Sec. 5.2).  LUT[k] = e^{-k} rounded to
// binary32; POLY coefficients as printed in Sec. 4, rounded to binary32.
constexpr float kLut[8] = {0x1p+0f,          0x1.78b564p-2f, 0x1.152aaap-3f, 0x1.97db0cp-5f,
                           0x1.2c155cp-6f,   0x1.b993fep-8f, 0x1.44e520p-9f, 0.0f};
constexpr float kC3 = -0x1.a3d70ap-4f;  // -0.1025
constexpr float kC2 = 0x1.d9b3d0p-2f;   //  0.4626
constexpr float kC1 = -0x1.fc01a4p-1f;  // -0.9922
constexpr float kC0 = 0x1.ffcb92p-1f;   //  0.9996
constexpr float kNr = 6.0f;

// Nearest integer (ties to even) of the exact product a*b, |a*b| < 2^22.
__device__ __forceinline__ int rne_mul(float a, float b) {
  return __float_as_int(__builtin_fmaf(a, b, kMagic)) - kMagicBits;
}

__device__ __forceinline__ float poly(float f) {
  return __builtin_fmaf(__builtin_fmaf(__builtin_fmaf(kC3, f, kC2), f, kC1), f, kC0);
}

// SAS of x = -y, y >= 0, with the table in LDS (8 floats, entry 7 = 0).
// Branch-free: y > 6 (x < n_r), y = +inf (a masked score) and y = NaN (a row
// with no visible key yet) all select the zero entry.
__device__ __forceinline__ int cvt_flr_i32(float x) {
  int r;
  asm("v_cvt_flr_i32_f32 %0, %1" : "=v"(r) : "v"(x));
  return r;
}

__device__ __forceinline__ float sas_y(float y, const float* lut) {
  const float yc = (y <= kNr) ? y : 7.0f;
  const float f = __builtin_amdgcn_fractf(yc);  // yc - floor(yc), exact
  return lut[cvt_flr_i32(yc)] * poly(f);
}

// Bits of fma(a, b, 1.5*2^23): the low byte is round-half-even(a*b) when
// 0 <= a*b < 256 (codes of Q(P~) and the like).
__device__ __forceinline__ int rne_bits(float a, float b) {
  return __float_as_int(__builtin_fmaf(a, b, kMagic));
}

// Low bytes of four dwords packed into one (two v_perm_b32).
__device__ __forceinline__ int pack_lo4(int x0, int x1, int x2, int x3) {
  const int t01 = (int)__builtin_amdgcn_perm((unsigned)x1, (unsigned)x0, 0x0c0c0400u);
  const int t23 = (int)__builtin_amdgcn_perm((unsigned)x3, (unsigned)x2, 0x04000c0cu);
  return t01 | t23;
}

// SAS with the table in registers (used where LDS is not set up).
__device__ __forceinline__ float sas_y_reg(float y) {
  const float yc = (y <= kNr) ? y : 7.0f;
  const float k = __builtin_floorf(yc);
  const float f = yc - k;
  const int idx = (int)k;
  float l = 0.0f;
#pragma unroll
  for (int i = 0; i < 7; ++i) l = (idx == i) ? kLut[i] : l;
  return l * poly(f);
}

// max(v, v of lane ^ 32): one v_permlane32_swap (gfx950) and one max.
__device__ __forceinline__ float max_xor32(float v) {
  const unsigned u = __float_as_uint(v);
  auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float add_xor32(float v) {
  const unsigned u = __float_as_uint(v);
  auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// max(v, v of lane ^ 16) within each 32-lane half: v_permlane16_swap.
__device__ __forceinline__ float max_xor16(float v) {
  const unsigned u = __float_as_uint(v);
  auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// max over the 16 lanes of a DPP row.
__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0xB1, 0xf, 0xf, false)));
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x4E, 0xf, 0xf, false)));
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x124, 0xf, 0xf, false)));
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x128, 0xf, 0xf, false)));
  return v;
}

// Maxima without NaN canonicalization (the compiler quiets both inputs of a
// max whose operands come from a lane exchange): one v_max_f32 for values
// that are never NaN, and the max of non-negative floats on their bits
// (integer order = float order), which also lets the DPP moves fuse into the
// max.
__device__ __forceinline__ float max_nn(float a, float b) {
  float r;
  asm("v_max_f32 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}

__device__ __forceinline__ float max_xor32_nn(float v) {
  const unsigned u = __float_as_uint(v);
  auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return max_nn(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float max_xor16_nn(float v) {
  const unsigned u = __float_as_uint(v);
  auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  return max_nn(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// max over the 64 lanes of a non-negative float (result in every lane)
__device__ __forceinline__ float wave_max_pos(float v) {
  int x = __float_as_int(v);
  x = max(x, __builtin_amdgcn_mov_dpp(x, 0xB1, 0xf, 0xf, true));
  x = max(x, __builtin_amdgcn_mov_dpp(x, 0x4E, 0xf, 0xf, true));
  x = max(x, __builtin_amdgcn_mov_dpp(x, 0x124, 0xf, 0xf, true));
  x = max(x, __builtin_amdgcn_mov_dpp(x, 0x128, 0xf, 0xf, true));
  auto r = __builtin_amdgcn_permlane16_swap((unsigned)x, (unsigned)x, false, false);
  x = max((int)r[0], (int)r[1]);
  r = __builtin_amdgcn_permlane32_swap((unsigned)x, (unsigned)x, false, false);
  return __int_as_float(max((int)r[0], (int)r[1]));
}

// max over the 64 lanes of the wave (result in every lane).
__device__ __forceinline__ float wave_max_fast(float v) {
  return max_xor32(max_xor16(row16_max(v)));
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, __shfl_xor(v, m));
  return v;
}

__device__ __forceinline__ int wave_max_i(int v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = max(v, __shfl_xor(v, m));
  return v;
}

__device__ __forceinline__ int wave_min_i(int v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = min(v, __shfl_xor(v, m));
  return v;
}

__device__ __forceinline__ v16i mfma32x32x32(v4i a, v4i b, v16i c) {
  return __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ v4i mfma16x16x64(v4i a, v4i b, v4i c) {
  return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
}

// Pack the low bytes of four ints (values -128..255) into one dword.
__device__ __forceinline__ int pack4(int a, int b, int c, int d) {
  return (a & 0xff) | ((b & 0xff) << 8) | ((c & 0xff) << 16) | ((int)((unsigned)d << 24));
}

}  // namespace turbo
