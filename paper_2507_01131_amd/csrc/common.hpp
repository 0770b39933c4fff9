// Shared device helpers for the gfx950 kernels of the CP tensor-product layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tdn {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kTile = 32;  // MFMA 32x32 output tile
constexpr int kNumXcd = 8;  // MI355X: 8 accelerator complex dies, blocks dealt round-robin

// One 32x32x2 fp32 MFMA.  Lane l supplies a = A[l%32][l/32] and
// b = B[l/32][l%32]; the 32x32 result is spread so that accumulator
// register v of lane l holds row acc_row(v, l/32), column l%32.
__device__ __forceinline__ f32x16 mfma32(float a, float b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ int acc_row(int v, int half) { return 8 * (v >> 2) + 4 * half + (v & 3); }

// One 16x16x4 fp32 MFMA.  Lane l supplies a = A[l%16][l/16] and
// b = B[l/16][l%16]; register i of lane l holds row 4(l/16) + i, column l%16.
__device__ __forceinline__ f32x4 mfma16f32(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float(uint32_t(h) << 16); }

template <typename T>
__device__ __forceinline__ float load_feat(const T* p);
template <>
__device__ __forceinline__ float load_feat<float>(const float* p) { return *p; }
template <>
__device__ __forceinline__ float load_feat<uint16_t>(const uint16_t* p) { return bf16_to_f32(*p); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
// Two floats rounded to bfloat16 (nearest even) and packed, a in the low
// half: one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2_rne(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{a, b}, bf16x2_t));
}
// Two-way half-precision split of a pair of floats, for fp32-accurate
// contractions on fp16 MFMA: v = hi + lo + r with hi = fp16(v) and
// lo = fp16(v - hi) (round to nearest even; v - hi is exact in fp32), so
// |r| <= 2^-22 |v| + 2^-25 (the second term from fp16 subnormals) for
// |v| < 2^15.  Callers scale each row by a power of two that puts its largest
// |v| in [2^13, 2^14), which makes the absolute term 2^-38 of that largest
// value.  Each part is packed as a pair, a in the low half: one
// v_cvt_pk_f16_f32 per part.
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_f16x2_rne(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{a, b}, f16x2_t));
}
__device__ __forceinline__ void split_f16x2_pair(float a, float b, uint32_t& hi, uint32_t& lo) {
  hi = pack_f16x2_rne(a, b);
  const f16x2_t h2 = __builtin_bit_cast(f16x2_t, hi);
  lo = pack_f16x2_rne(a - float(h2[0]), b - float(h2[1]));
}
// Power-of-two exponent e with max_abs * 2^-e in [2^13, 2^14) (0 for 0 or
// non-finite input), clamped so that 2^e and 2^-e are normal floats.
__device__ __forceinline__ int f16_split_exponent(float max_abs) {
  if (!(max_abs > 0.f) || !(max_abs < 3.0e38f)) return 0;
  int E;
  (void)frexpf(max_abs, &E);  // max_abs = m 2^E, m in [0.5, 1)
  const int e = E - 14;
  return e < -125 ? -125 : (e > 125 ? 125 : e);
}

// A 32x32 MFMA accumulator tile as the K operand of a 32x32x16 step: K-step
// q (0, 1) of lane half h takes the rows held in accumulator registers
// 8q .. 8q+7, i.e. row acc_krow(q, h, i) for element i = 0..7.  The other
// operand is laid out with the same row order.
__host__ __device__ constexpr int acc_krow(int q, int h, int i) { return 16 * q + 8 * (i / 4) + 4 * h + (i % 4); }

// Blocks of a 1-D grid are dealt to the XCDs round-robin (block b runs on XCD
// b % 8).  Remap so that each XCD walks one contiguous range of logical work
// items: neighbouring destination nodes share source nodes, and then share
// that XCD's L2.  The map is a bijection on [0, total).
__device__ __forceinline__ int xcd_remap(int b, int total) {
  const int per = total / kNumXcd, rem = total % kNumXcd;
  const int xcd = b % kNumXcd, j = b / kNumXcd;
  return xcd < rem ? xcd * (per + 1) + j : rem * (per + 1) + (xcd - rem) * per + j;
}

}  // namespace tdn
