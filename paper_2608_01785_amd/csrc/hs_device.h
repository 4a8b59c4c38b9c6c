// Device-side helpers shared by the gfx950 kernels: bf16 vectors, MFMA
// wrappers, LDS swizzles and the XCD-aware work-group remap.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hs {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;
constexpr int kNumXcd = 8;

// 32x32x16 bf16 MFMA, fp32 accumulate.
//   A operand: lane l holds A[i = l % 32][k = 8 (l / 32) + 0..7]
//   B operand: lane l holds B[k = 8 (l / 32) + 0..7][j = l % 32]
//   D:         lane l, register r holds D[i = 8 (r / 4) + 4 (l / 32) + r % 4][j = l % 32]
__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float bf2f(uint16_t h) { return __uint_as_float(uint32_t(h) << 16); }

__device__ __forceinline__ uint16_t f2bf(float f) {
  __bf16 b = (__bf16)f;  // round to nearest even (v_cvt_pk_bf16_f32 on gfx950)
  return __builtin_bit_cast(uint16_t, b);
}

__device__ __forceinline__ uint32_t pack2bf(float lo, float hi) {
  return uint32_t(f2bf(lo)) | (uint32_t(f2bf(hi)) << 16);
}

__device__ __forceinline__ bf16x8 as_bf16x8(const u32x4& v) { return __builtin_bit_cast(bf16x8, v); }

// Store 4 consecutive bf16 values (8 bytes, 8-byte aligned).
__device__ __forceinline__ void store_bf16x4(uint16_t* p, float a, float b, float c, float d) {
  u32x2 v;
  v.x = pack2bf(a, b);
  v.y = pack2bf(c, d);
  *reinterpret_cast<u32x2*>(p) = v;
}

__device__ __forceinline__ void load_bf16x4(const uint16_t* p, float out[4]) {
  u32x2 v = *reinterpret_cast<const u32x2*>(p);
  out[0] = __uint_as_float(v.x << 16);
  out[1] = __uint_as_float(v.x & 0xffff0000u);
  out[2] = __uint_as_float(v.y << 16);
  out[3] = __uint_as_float(v.y & 0xffff0000u);
}

// Work-groups of a launch are handed to the 8 XCDs round-robin (block b runs
// on XCD b % 8).  Remap so that each XCD processes a contiguous range of
// logical work items, which then share operands in that XCD's L2.
__device__ __forceinline__ int xcd_remap(int bid, int nblocks) {
  if (nblocks % kNumXcd != 0) return bid;
  const int per = nblocks / kNumXcd;
  return (bid % kNumXcd) * per + bid / kNumXcd;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

}  // namespace hs
