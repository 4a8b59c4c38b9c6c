// Device-side helpers shared by the gfx950 kernels: bf16 vectors, MFMA
// wrappers, LDS swizzles and the XCD-aware work-group remap.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hs {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;
constexpr int kNumXcd = 8;
constexpr float kF16Max = 65504.0f;

// 32x32x16 fp16 MFMA, fp32 accumulate.  Operands are 8 packed fp16 values.
//   A operand: lane l holds A[i = l % 32][k = 8 (l / 32) + 0..7]
//   B operand: lane l holds B[k = 8 (l / 32) + 0..7][j = l % 32]
//   D:         lane l, register r holds D[i = 8 (r / 4) + 4 (l / 32) + r % 4][j = l % 32]
__device__ __forceinline__ f32x16 mfma32(const u32x4& a, const u32x4& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c,
                                                0, 0, 0);
}

__device__ __forceinline__ float bf2f(uint16_t h) { return __uint_as_float(uint32_t(h) << 16); }

__device__ __forceinline__ float h2f(uint16_t h) { return float(__builtin_bit_cast(_Float16, h)); }

// fp32 -> fp16, round to nearest even, saturated to the finite range.
__device__ __forceinline__ uint16_t f2h(float f) {
  f = fminf(fmaxf(f, -kF16Max), kF16Max);
  return __builtin_bit_cast(uint16_t, (_Float16)f);
}

// Two fp32 values -> two fp16 values as f2h does, with one packed conversion.
__device__ __forceinline__ uint32_t pack2h(float lo, float hi) {
  typedef float f2 __attribute__((ext_vector_type(2)));
  typedef _Float16 h2 __attribute__((ext_vector_type(2)));
  const f2 v = {fminf(fmaxf(lo, -kF16Max), kF16Max), fminf(fmaxf(hi, -kF16Max), kF16Max)};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, h2));
}

// 2^x with the hardware instruction alone (about 1 ulp; results below the
// normal range flush to zero, which softmax weights can afford).
__device__ __forceinline__ float exp2_raw(float x) { return __builtin_amdgcn_exp2f(x); }

// Two bf16 values (one 32-bit word) -> two fp16 values.  Exact for
// magnitudes in [2^-14, 65504]; smaller values become fp16 subnormals
// (absolute error below 2^-24).  Round-toward-zero conversion is used because
// it is a single packed instruction and is exact wherever fp16 can hold the
// bf16 value.
__device__ __forceinline__ uint32_t bf2x_to_h2x(uint32_t u) {
  const float lo = __uint_as_float(u << 16);
  const float hi = __uint_as_float(u & 0xffff0000u);
  return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pkrtz(lo, hi));
}

__device__ __forceinline__ u32x4 bf8_to_h8(const u32x4& v) {
  u32x4 r;
  r.x = bf2x_to_h2x(v.x);
  r.y = bf2x_to_h2x(v.y);
  r.z = bf2x_to_h2x(v.z);
  r.w = bf2x_to_h2x(v.w);
  return r;
}

// Store 4 consecutive fp16 values (8 bytes, 8-byte aligned).
__device__ __forceinline__ void store_h4(uint16_t* p, float a, float b, float c, float d) {
  u32x2 v;
  v.x = pack2h(a, b);
  v.y = pack2h(c, d);
  *reinterpret_cast<u32x2*>(p) = v;
}

// Two groups of four fp16 outputs of one row in the 32x32 MFMA accumulator
// layout: lane r + 32 h holds columns 4h .. 4h + 3 of group `lo` (columns
// 0..7 of a 16-column run) and of group `hi` (columns 8..15).  One permlane32
// swap per dword, which exchanges lanes 32..63 of its first operand with
// lanes 0..31 of its second, leaves all eight columns of `lo` in the low lane
// and all eight of `hi` in the high one, as eight packed fp16 values: lane
// r + 32 h then owns columns 8h .. 8h + 7 of the run.  Both lanes of a row
// must be active.
__device__ __forceinline__ u32x4 swap_h8(const float (&lo)[4], const float (&hi)[4]) {
  const uint32_t a[2] = {pack2h(lo[0], lo[1]), pack2h(lo[2], lo[3])};
  const uint32_t b[2] = {pack2h(hi[0], hi[1]), pack2h(hi[2], hi[3])};
  u32x4 v;
#pragma unroll
  for (int d = 0; d < 2; ++d) {
    const auto s = __builtin_amdgcn_permlane32_swap(a[d], b[d], false, false);
    v[d] = s[0];
    v[2 + d] = s[1];
  }
  return v;
}

// swap_h8 stored row-major: the run starts at p, so each lane writes 16
// contiguous bytes at p + 8h and the two lanes of a row cover 32.
__device__ __forceinline__ void store_h8_pair(uint16_t* p, int h, const float (&lo)[4], const float (&hi)[4]) {
  *reinterpret_cast<u32x4*>(p + 8 * h) = swap_h8(lo, hi);
}

// Element offset of activation (m, k): row-major with row stride ld, or, when
// k8_rows > 0, k-group-major ((k / 8) * k8_rows + m) * 8 + k % 8, the layout
// in which a 32-row MFMA operand fragment of 8 k values per lane is one
// contiguous 512-byte run.
__device__ __forceinline__ int64_t act_index(int m, int k, int ld, int k8_rows) {
  return k8_rows ? (int64_t(k >> 3) * k8_rows + m) * 8 + (k & 7) : int64_t(m) * ld + k;
}

// MFMA row i of a 32-key subtile reads key perm32(i): bits 2 and 3 swapped.
__device__ __forceinline__ int perm32(int i) {
  return (i & ~12) | ((i >> 1) & 4) | ((i << 1) & 8);
}

// Memory accesses whose data another block of the same launch reads or wrote
// (DEV = true): device-scope relaxed atomics, which write through to, and read
// from, the device-coherent level instead of an XCD's private L2.  With
// DEV = false they are ordinary accesses.
template <bool DEV>
__device__ __forceinline__ void st_u64(void* p, uint64_t v) {
  if constexpr (DEV)
    __hip_atomic_store(static_cast<uint64_t*>(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  else
    *static_cast<uint64_t*>(p) = v;
}
template <bool DEV>
__device__ __forceinline__ uint64_t ld_u64(const void* p) {
  if constexpr (DEV)
    return __hip_atomic_load(static_cast<const uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  else
    return *static_cast<const uint64_t*>(p);
}
template <bool DEV>
__device__ __forceinline__ void st_u16(uint16_t* p, uint16_t v) {
  if constexpr (DEV)
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  else
    *p = v;
}
template <bool DEV>
__device__ __forceinline__ void st_f32(float* p, float v) {
  if constexpr (DEV)
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  else
    *p = v;
}
template <bool DEV>
__device__ __forceinline__ float ld_f32(const float* p) {
  if constexpr (DEV)
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  else
    return *p;
}
template <bool DEV>
__device__ __forceinline__ u32x4 ld_u32x4(const void* p) {
  if constexpr (DEV) {
    const uint64_t lo = ld_u64<true>(p), hi = ld_u64<true>(static_cast<const uint8_t*>(p) + 8);
    u32x4 r;
    r[0] = uint32_t(lo);
    r[1] = uint32_t(lo >> 32);
    r[2] = uint32_t(hi);
    r[3] = uint32_t(hi >> 32);
    return r;
  } else {
    return *static_cast<const u32x4*>(p);
  }
}
template <bool DEV>
__device__ __forceinline__ void st_f32x4(float* p, f32x4 v) {
  if constexpr (DEV) {
    st_u64<true>(p, uint64_t(__float_as_uint(v[0])) | (uint64_t(__float_as_uint(v[1])) << 32));
    st_u64<true>(p + 2, uint64_t(__float_as_uint(v[2])) | (uint64_t(__float_as_uint(v[3])) << 32));
  } else {
    *reinterpret_cast<f32x4*>(p) = v;
  }
}
template <bool DEV>
__device__ __forceinline__ f32x4 ld_f32x4(const float* p) {
  if constexpr (DEV) {
    const uint64_t lo = ld_u64<true>(p), hi = ld_u64<true>(p + 2);
    return f32x4{__uint_as_float(uint32_t(lo)), __uint_as_float(uint32_t(lo >> 32)), __uint_as_float(uint32_t(hi)),
                 __uint_as_float(uint32_t(hi >> 32))};
  } else {
    return *reinterpret_cast<const f32x4*>(p);
  }
}
template <bool DEV>
__device__ __forceinline__ void st_h4(uint16_t* p, float a, float b, float c, float d) {
  st_u64<DEV>(p, uint64_t(pack2h(a, b)) | (uint64_t(pack2h(c, d)) << 32));
}

__device__ __forceinline__ void load_bf16x4(const uint16_t* p, float out[4]) {
  u32x2 v = *reinterpret_cast<const u32x2*>(p);
  out[0] = __uint_as_float(v.x << 16);
  out[1] = __uint_as_float(v.x & 0xffff0000u);
  out[2] = __uint_as_float(v.y << 16);
  out[3] = __uint_as_float(v.y & 0xffff0000u);
}

// Two packed fp16 values -> floats.
__device__ __forceinline__ void h2x_to_f(uint32_t u, float& lo, float& hi) {
  lo = h2f(uint16_t(u & 0xffffu));
  hi = h2f(uint16_t(u >> 16));
}

// Launch clock record (timing mode only): the first lane of block 0 reads the
// shader-clock counter (s_memtime, counts core clock cycles) and the
// constant-rate counter (s_memrealtime) at entry and exit and stores the four
// values with one vector store, so the host can derive the sustained clock.
struct LaunchClock {
  uint64_t c0 = 0, w0 = 0;
  __device__ __forceinline__ void begin(const uint64_t* out) {
    if (out && blockIdx.x == 0 && threadIdx.x == 0) {
      c0 = __builtin_amdgcn_s_memtime();
      w0 = __builtin_amdgcn_s_memrealtime();
    }
  }
  __device__ __forceinline__ void end(uint64_t* out) const {
    if (out && blockIdx.x == 0 && threadIdx.x == 0) {
      const uint64_t c1 = __builtin_amdgcn_s_memtime();
      const uint64_t w1 = __builtin_amdgcn_s_memrealtime();
      out[0] = c0;
      out[1] = w0;
      out[2] = c1;
      out[3] = w1;
    }
  }
};

// Work-groups of a launch are handed to the 8 XCDs round-robin (block b runs
// on XCD b % 8).  Remap so that each XCD processes a contiguous range of
// logical work items, which then share operands in that XCD's L2.
__device__ __forceinline__ int xcd_remap(int bid, int nblocks) {
  if (nblocks % kNumXcd != 0) return bid;
  const int per = nblocks / kNumXcd;
  return (bid % kNumXcd) * per + bid / kNumXcd;
}

// RoPE position of row m for rotary pair j (plain or sectioned multimodal).
template <typename Args>
__device__ __forceinline__ int rope_pos(const Args& a, int m, int j) {
  const int c = int(j >= a.sec1) + int(j >= a.sec2);
  return a.pos[c * a.pos_stride + m];
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
