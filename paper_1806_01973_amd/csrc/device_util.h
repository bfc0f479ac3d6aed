// Device-side helpers shared by the gfx950 kernels of libpinsage.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pinsage {

constexpr int kWave = 64;

// Philox4x32-10 block function (Salmon et al., SC'11): ten rounds of two
// 32x32->64 multiplies whose halves are mixed with the other counter words and
// the key; the key advances by the Weyl constants between rounds.
__device__ __forceinline__ uint4 philox4x32_10(uint4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint32_t lo0 = c.x * 0xD2511F53u;
    const uint32_t hi0 = __umulhi(c.x, 0xD2511F53u);
    const uint32_t lo1 = c.z * 0xCD9E8D57u;
    const uint32_t hi1 = __umulhi(c.z, 0xCD9E8D57u);
    c = make_uint4(hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0);
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return c;
}

// bf16 storage is a raw 16-bit pattern (upper half of an fp32).
__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(((uint32_t)b) << 16);
}

// fp32 -> bf16, round to nearest, ties to even (NaN stays a quiet NaN).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// Two fp32 values to a packed bf16 pair (low half = lo) with the gfx950
// conversion instruction: round to nearest, ties to even, like f32_to_bf16.
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const bf16x2_t v = __builtin_convertvector((f32x2_t){lo, hi}, bf16x2_t);
  return __builtin_bit_cast(uint32_t, v);
}

// Orders LDS accesses of one wavefront across its lanes (all lanes of a wave
// execute in lockstep; this keeps the compiler from reordering LDS traffic
// across the point and waits for outstanding LDS operations).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// ---- cross-lane exchange through DPP (VALU, no LDS traffic) ----------------
// Controls (gfx9 encoding): quad_perm 0xB1 / 0x4E read lane ^ 1 / lane ^ 2;
// row_ror:n (0x120 + n) reads lane (i - n) mod 16 within each row of 16 lanes;
// row_shr:n (0x110 + n) reads lane i - n within the row (lanes without a
// source keep `old`); row_bcast:15 / :31 (0x142 / 0x143) read lane 15 of the
// previous row / lane 31.
template <int CTRL, int ROW_MASK = 0xF>
__device__ __forceinline__ int dpp(int old, int v) {
  return __builtin_amdgcn_update_dpp(old, v, CTRL, ROW_MASK, 0xF, false);
}

// Value held by lane (lane ^ M), M a power of two below 64.
template <int M>
__device__ __forceinline__ uint32_t lane_xor(uint32_t v, int lane) {
  const int x = (int)v;
  if constexpr (M == 1) {
    return (uint32_t)dpp<0xB1>(x, x);
  } else if constexpr (M == 2) {
    return (uint32_t)dpp<0x4E>(x, x);
  } else if constexpr (M == 4) {
    const int up = dpp<0x12C>(x, x);    // lane i + 4 (row_ror:12)
    const int down = dpp<0x124>(x, x);  // lane i - 4 (row_ror:4)
    return (uint32_t)((lane & 4) ? down : up);
  } else if constexpr (M == 8) {
    return (uint32_t)dpp<0x128>(x, x);  // row_ror:8
  } else if constexpr (M == 16) {
    return (uint32_t)__builtin_amdgcn_ds_swizzle(x, 0x1F | (16 << 10));  // bit-mode xor 16
  } else {
    return (uint32_t)__shfl_xor(x, M);
  }
}

// Inclusive scans over the 64 lanes: Hillis-Steele inside rows of 16, then the
// row totals are carried across rows with the two row broadcasts.
__device__ __forceinline__ int wave_inclusive_sum(int v, int /*lane*/) {
  v += dpp<0x111>(0, v);
  v += dpp<0x112>(0, v);
  v += dpp<0x114>(0, v);
  v += dpp<0x118>(0, v);
  v += dpp<0x142, 0xA>(0, v);
  v += dpp<0x143, 0xC>(0, v);
  return v;
}

__device__ __forceinline__ int imax(int a, int b) { return a > b ? a : b; }

// Identity -1 (the values scanned here are >= -1).
__device__ __forceinline__ int wave_inclusive_max(int v, int /*lane*/) {
  v = imax(v, dpp<0x111>(-1, v));
  v = imax(v, dpp<0x112>(-1, v));
  v = imax(v, dpp<0x114>(-1, v));
  v = imax(v, dpp<0x118>(-1, v));
  v = imax(v, dpp<0x142, 0xA>(-1, v));
  v = imax(v, dpp<0x143, 0xC>(-1, v));
  return v;
}

// Butterfly sum: every lane ends with the same total, added in a fixed order.
__device__ __forceinline__ float wave_sum_f32(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Wave-wide max / sum of values >= -1 (resp. any int), same on every lane.
__device__ __forceinline__ int wave_max_i32(int v) {
  return __builtin_amdgcn_readlane(wave_inclusive_max(v, 0), 63);
}

__device__ __forceinline__ int wave_sum_i32(int v) {
  return __builtin_amdgcn_readlane(wave_inclusive_sum(v, 0), 63);
}

}  // namespace pinsage
