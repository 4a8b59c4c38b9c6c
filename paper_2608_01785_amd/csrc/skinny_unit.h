// One block's unit of the skinny (decode-sized) fp16 MFMA GEMM, shared by the
// standalone skinny kernel and the persistent decode-layer kernel.
//
// Decode re-reads every weight for a handful of rows, so the unit streams W
// rather than reusing it: a block owns a thin strip of weight rows (32, or 64
// when the epilogue needs RoPE or gate/up pairs) and all M rows, and walks K
// in 64-wide stages copied buffer -> LDS by the load unit through a ring.
// The four waves split every stage's K: wave w multiplies the 16-wide slice w,
// so no wave waits on another until the end, where partial accumulators are
// summed through LDS and the fused epilogues run (residual add into fp32,
// SwiGLU, or RoPE + key/value store).  A K split publishes fp32 partial sums;
// the last split of a strip to arrive adds them in split order.
//
// Weights are bf16 row-major or prepared fp16 panel-major ([K / 32][N][32]).
// The weight strip is the MFMA A operand and activation rows the B operand, so
// each lane of a 32x32 accumulator owns one activation row and 4 consecutive
// output columns per register group.
#pragma once

#include "hs_device.h"
#include "hs_kernels.h"

namespace hs {
namespace skinny {

constexpr int BK = kSkinnyBK;           // K per stage
constexpr int kRowBytes = BK * 2;       // 128 bytes, 8 chunks of 16
constexpr int kMaxStages = 8;
constexpr int kLdsBytes = 160 * 1024;
constexpr int kThreads = 256;
constexpr int kDeviceScope = 16;        // buffer cache-policy bit sc1: device-coherent access

using lds_ptr_t = __attribute__((address_space(3))) void*;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, 0x00020000);
}

__device__ __forceinline__ void barrier_nofence() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // this wave's LDS reads are done
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

__device__ __forceinline__ float silu(float z) { return z / (1.0f + __expf(-z)); }

// Wait until at most n stages of this wave's copies are outstanding, with L
// copies per stage.
template <int L>
__device__ __forceinline__ void wait_stages(int n) {
  switch (n) {
#define HS_CASE(k)                                                           \
  case k:                                                                    \
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"((k * L) < 63 ? (k * L) : 63) : "memory"); \
    break;
    HS_CASE(0) HS_CASE(1) HS_CASE(2) HS_CASE(3) HS_CASE(4) HS_CASE(5)
    default:
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"((6 * L) < 63 ? (6 * L) : 63) : "memory");
      break;
#undef HS_CASE
  }
}

// 16-byte chunk c of a 64-byte panel row r sits at physical chunk c ^ swz4(r).
__device__ __forceinline__ int swz4(int r) { return (r >> 1) & 3; }

// Weight row held in row r of strip `tile` (NR rows per strip).
template <int EPI, int NR>
__device__ __forceinline__ uint32_t strip_row(int tile, int r, int ffn) {
  if constexpr (EPI == EPI_SWIGLU) {
    return uint32_t((r >> 5) * ffn + tile * 32 + (r & 31));  // [gate 32 | up 32]
  } else {
    return uint32_t(tile * NR + r);
  }
}

template <int EPI, int DH, bool W_F16, int NS, int MT, int ST>
struct SkinnyShape {
  static constexpr int NR = 32 * NS;
  static constexpr int MR = 32 * MT;
  static constexpr int STAGE = (NR + MR) * kRowBytes;
  static constexpr int kStages = (kLdsBytes / STAGE) < ST ? (kLdsBytes / STAGE) : ST;
  static constexpr int RED = 4 * NS * MT * 16 * 64 * 4;
  static constexpr int SMEM = (kStages * STAGE > RED + 16) ? kStages * STAGE : RED + 16;
};

// One weight strip (`tile`) and one K split (`ks`) of a skinny GEMM, by one
// block of kThreads threads, in LDS `smem` (SkinnyShape::SMEM bytes, 1 KB
// aligned).  DEV: the activations, residual and outputs are shared with other
// blocks of the same launch (device-scope accesses).
template <int EPI, int DH, bool W_F16, int NS, int MT, int ST, bool DEV>
__device__ __forceinline__ void skinny_unit(const GemmArgs& a, int tile, int ks, uint8_t* smem) {
  constexpr int NR = 32 * NS;                 // weight rows per block
  constexpr int MR = 32 * MT;                 // activation rows covered
  constexpr int WBYTES = NR * kRowBytes;
  constexpr int XBYTES = MR * kRowBytes;
  constexpr int STAGE = WBYTES + XBYTES;
  constexpr int WCOPIES = NR / 8 / 4;         // copies per wave per stage (8 rows each)
  constexpr int XCOPIES = MR / 8 / 4;
  constexpr int L = WCOPIES + XCOPIES;
  constexpr int kStages = (kLdsBytes / STAGE) < ST ? (kLdsBytes / STAGE) : ST;
  constexpr int RED = 4 * NS * MT * 16 * 64 * 4;  // cross-wave reduction buffer
  constexpr int SMEM = (kStages * STAGE > RED + 16) ? kStages * STAGE : RED + 16;
  static_assert(NR % 32 == 0 && MR % 32 == 0, "tile shape");
  static_assert(SMEM <= kLdsBytes, "LDS");

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int fr = lane & 31, fh = lane >> 5;
  const int n_split = a.n_split;
  // Folded RMSNorm: this lane's row's partial sums of squares, loaded now and
  // summed in the epilogue (wave w owns rows 32 w .. 32 w + 31 there).  Rows
  // past M fall outside the buffer range and read zero.
  constexpr int kPre = (EPI == EPI_RESID) ? 1 : kSkinnyMaxNormParts / 4;
  u32x4 pre[kPre];
  const bool want_rs = EPI != EPI_RESID && a.row_sumsq && wave < MT;
  if (want_rs) {
    const __amdgpu_buffer_rsrc_t pr = make_rsrc(a.row_sumsq, uint32_t(a.M) * a.row_parts * 4);
    const uint32_t row_off = uint32_t((wave * 32 + fr) * a.row_parts) * 4;
#pragma unroll
    for (int u = 0; u < kPre; ++u)
      if (4 * u < a.row_parts)
        pre[u] = __builtin_amdgcn_raw_buffer_load_b128(pr, row_off + uint32_t(u * 16), 0, DEV ? kDeviceScope : 0);
  }
  const int kt0 = ks * a.k_per_split;
  const int KT = min(a.K / BK - kt0, a.k_per_split);  // stages of this split
  const uint32_t row_bytes = uint32_t(a.K) * 2;

  const uint32_t w_rows = (EPI == EPI_SWIGLU) ? uint32_t(2 * a.ffn) : uint32_t(a.n_tiles_n * 256);
  const __amdgpu_buffer_rsrc_t wres = make_rsrc(a.W, w_rows * row_bytes);
  const __amdgpu_buffer_rsrc_t xres = make_rsrc(a.A, uint32_t(a.M) * row_bytes);

  // Activation copies: one wave instruction fills 8 rows of 128 bytes; lane i
  // lands at row i / 8, physical chunk i % 8 = logical chunk (i % 8) ^ (row % 8).
  const int sub = lane >> 3;
  const int chunk = (lane & 7) ^ sub;
  // Weight copies.  Row-major bf16: as the activations.  Panel-major fp16
  // ([K / 32][N][32]): a stage is two 32-wide panels, stored in LDS as
  // [panel][NR rows][64 bytes]; one instruction fills 16 rows of one panel,
  // lane i at row i / 4, physical chunk i % 4 = logical (i % 4) ^ swz4(row).
  const int psub = lane >> 2;
  const int pchunk = (lane & 3) ^ swz4(psub);
  // Fixed extents: arrays sized by the template's constants and captured by
  // the lambda below make the host pass drop the kernel's launch stub.
  static_assert(WCOPIES <= 2 && XCOPIES <= 4, "copy slots");
  uint32_t w_off[2], x_off[4];
  int w_panel[2];
#pragma unroll
  for (int c = 0; c < WCOPIES; ++c) {
    const int q = wave * WCOPIES + c;
    if constexpr (W_F16) {
      w_panel[c] = q / (NR / 16);
      w_off[c] = strip_row<EPI, NR>(tile, (q % (NR / 16)) * 16 + psub, a.ffn) * 64 + pchunk * 16;
    } else {
      w_panel[c] = 0;
      w_off[c] = strip_row<EPI, NR>(tile, q * 8 + sub, a.ffn) * row_bytes + chunk * 16;
    }
  }
#pragma unroll
  for (int c = 0; c < XCOPIES; ++c) x_off[c] = uint32_t((wave * XCOPIES + c) * 8 + sub) * row_bytes + chunk * 16;
  const uint32_t panel_bytes = w_rows * 64;

  auto issue = [&](int kt, int buf) {
    const int koff = (kt0 + kt) * kRowBytes;
    uint8_t* base = smem + buf * STAGE;
#pragma unroll
    for (int c = 0; c < WCOPIES; ++c) {
      // Both layouts put copy q at byte q * 1 KB of the stage's weight area.
      const int q = wave * WCOPIES + c;
      const uint32_t soff = W_F16 ? (2 * (kt0 + kt) + w_panel[c]) * panel_bytes : uint32_t(koff);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(wres, (lds_ptr_t)(base + q * 1024), 16, w_off[c], soff, 0, 0);
    }
#pragma unroll
    for (int c = 0; c < XCOPIES; ++c)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(xres,
                                               (lds_ptr_t)(base + WBYTES + (wave * XCOPIES + c) * 8 * kRowBytes),
                                               16, x_off[c], koff, 0, DEV ? kDeviceScope : 0);
  };

  f32x16 acc[NS][MT];
#pragma unroll
  for (int i = 0; i < NS; ++i)
#pragma unroll
    for (int j = 0; j < MT; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

#pragma unroll
  for (int st = 0; st < kStages - 1; ++st)
    if (st < KT) issue(st, st);

  const int phys = (2 * wave + fh) ^ (fr & 7);  // this wave's 16-wide K slice
  // Panel-major weights: slice w is chunks 2 (w % 2) + fh of panel w / 2.
  const int pphys = (2 * (wave & 1) + fh) ^ swz4(fr);
  const int pbase = (wave >> 1) * NR * 64;
  int buf = 0;
  for (int kt = 0; kt < KT; ++kt) {
    wait_stages<L>(min(kStages - 2, KT - 1 - kt));
    barrier_nofence();
    if (kt + kStages - 1 < KT) issue(kt + kStages - 1, buf == 0 ? kStages - 1 : buf - 1);
    const uint8_t* base = smem + buf * STAGE;
    u32x4 fw[NS], fx[MT];
#pragma unroll
    for (int i = 0; i < NS; ++i)
      fw[i] = W_F16 ? *reinterpret_cast<const u32x4*>(base + pbase + (i * 32 + fr) * 64 + pphys * 16)
                    : *reinterpret_cast<const u32x4*>(base + (i * 32 + fr) * kRowBytes + phys * 16);
#pragma unroll
    for (int j = 0; j < MT; ++j)
      fx[j] = *reinterpret_cast<const u32x4*>(base + WBYTES + (j * 32 + fr) * kRowBytes + phys * 16);
#pragma unroll
    for (int i = 0; i < NS; ++i) {
      const u32x4 wh = W_F16 ? fw[i] : bf8_to_h8(fw[i]);
#pragma unroll
      for (int j = 0; j < MT; ++j) acc[i][j] = mfma32(wh, fx[j], acc[i][j]);
    }
    buf = (buf == kStages - 1) ? 0 : buf + 1;
  }

  // Sum the four waves' partial accumulators through LDS; wave w then owns
  // row subtile j = w (MT <= 4).
  __syncthreads();
  float* red = reinterpret_cast<float*>(smem);
#pragma unroll
  for (int i = 0; i < NS; ++i)
#pragma unroll
    for (int j = 0; j < MT; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) red[(((wave * NS + i) * MT + j) * 16 + r) * 64 + lane] = acc[i][j][r];
  __syncthreads();
  const int j = wave;
  const bool owner = j < MT;
  f32x16 c[NS];
#pragma unroll
  for (int i = 0; i < NS; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      float v = 0.0f;
      if (owner) {
#pragma unroll
        for (int w = 0; w < 4; ++w) v += red[(((w * NS + i) * MT + j) * 16 + r) * 64 + lane];
      }
      c[i][r] = v;
    }

  if (n_split > 1) {
    // Publish this split's sums; the last split of the strip to arrive adds
    // all splits in split order (the same order whoever arrives last) and
    // runs the epilogue.  Partial sums move with device-scope (sc1) vector
    // accesses, which write through to and read from the coherent level, so
    // no agent-scope fence (a full L2 write-back and invalidate) is needed.
    constexpr int IMG = NS * MT * 16 * 64;  // floats per split image: [i][j][lane][16]
    const __amdgpu_buffer_rsrc_t pres =
        make_rsrc(a.part + size_t(tile) * n_split * IMG, uint32_t(n_split) * IMG * 4);
    if (owner) {
#pragma unroll
      for (int i = 0; i < NS; ++i)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const f32x4 v = {c[i][4 * q], c[i][4 * q + 1], c[i][4 * q + 2], c[i][4 * q + 3]};
          const uint32_t off = uint32_t(((ks * NS + i) * MT + j) * 1024 + lane * 16 + 4 * q) * 4;
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), pres, off, 0, kDeviceScope);
        }
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // stores complete before the arrival count
    __syncthreads();
    int* last = reinterpret_cast<int*>(smem + SMEM - 16);  // past the reduction buffer
    if (tid == 0) {
      const int arrived = atomicAdd(a.counters + tile, 1);
      *last = arrived == n_split - 1;
      if (*last) __hip_atomic_store(a.counters + tile, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
    if (!*last) return;
    // All threads add the split images (every load in flight at once), then
    // the owners pick their registers up from LDS.
    f32x4* red4 = reinterpret_cast<f32x4*>(smem);
    for (int e = tid; e < IMG / 4; e += kThreads) {
      // Splits past n_split lie outside the buffer resource and read zero.
      u32x4 x[kSkinnyMaxSplits];
#pragma unroll
      for (int sp = 0; sp < kSkinnyMaxSplits; ++sp)
        x[sp] = __builtin_amdgcn_raw_buffer_load_b128(pres, uint32_t((sp * IMG + 4 * e) * 4), 0, kDeviceScope);
      f32x4 v = __builtin_bit_cast(f32x4, x[0]);
#pragma unroll
      for (int sp = 1; sp < kSkinnyMaxSplits; ++sp) v += __builtin_bit_cast(f32x4, x[sp]);
      red4[e] = v;
    }
    __syncthreads();
    if (owner) {
#pragma unroll
      for (int i = 0; i < NS; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) c[i][r] = reinterpret_cast<const float*>(red4)[((i * MT + j) * 64 + lane) * 16 + r];
    }
  }

  const int m = j * 32 + fr;
  if constexpr (EPI == EPI_RESID) {
    const int strips = a.n_tiles_n * 256 / NR;
    if (owner && m < a.M) {
      float* orow = a.out_f32 + int64_t(m) * a.ldo;
      float ss = 0.0f;
#pragma unroll
      for (int i = 0; i < NS; ++i)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int n = tile * NR + i * 32 + 8 * g + 4 * fh;
          f32x4 v = {c[i][4 * g], c[i][4 * g + 1], c[i][4 * g + 2], c[i][4 * g + 3]};
          if (a.resid_f32) {
            v += ld_f32x4<DEV>(a.resid_f32 + int64_t(m) * a.ldo + n);
          } else {
            float r4[4];
            load_bf16x4(a.resid + int64_t(m) * a.ldo + n, r4);
            v[0] += r4[0];
            v[1] += r4[1];
            v[2] += r4[2];
            v[3] += r4[3];
          }
          st_f32x4<DEV>(orow + n, v);
          ss += v[0] * v[0] + v[1] * v[1] + v[2] * v[2] + v[3] * v[3];
          if (a.scaled_out) {
            float gm[4];
            load_bf16x4(a.gain + n, gm);
            st_h4<DEV>(a.scaled_out + int64_t(m) * a.ldo + n, v[0] * gm[0], v[1] * gm[1], v[2] * gm[2], v[3] * gm[3]);
          }
        }
      if (a.sumsq_out) {
        // The lane pair (fh = 0, 1) holds this row's NR columns of the strip.
        ss += __shfl_xor(ss, 32, 64);
        if (fh == 0) st_f32<DEV>(a.sumsq_out + int64_t(m) * strips + tile, ss);
      }
    }
    return;
  } else {
    if (!owner || m >= a.M) return;
    if (want_rs) {
      float sum = 0.0f;
#pragma unroll
      for (int u = 0; u < kPre; ++u) {
        if (4 * u >= a.row_parts) break;
        const f32x4 f = __builtin_bit_cast(f32x4, pre[u]);
        sum += f[0];
        sum += f[1];
        sum += f[2];
        sum += f[3];
      }
      const float rs = rsqrtf(sum / float(a.K) + a.eps);
#pragma unroll
      for (int i = 0; i < NS; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) c[i][r] *= rs;
    }
  }
  if constexpr (EPI == EPI_SWIGLU) {
    static_assert(EPI != EPI_SWIGLU || NS == 2, "gate/up strips hold 32 + 32 rows");
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      float v[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = silu(c[0][4 * g + e]) * c[1][4 * g + e];
      st_h4<DEV>(a.out + int64_t(m) * a.ldo + tile * 32 + 8 * g + 4 * fh, v[0], v[1], v[2], v[3]);
    }
  } else {  // EPI_QKV: the strip is one 64-wide head
    static_assert(EPI != EPI_QKV || (NS == 2 && DH == 64), "QKV strips are one 64-wide head");
    const int head = tile;
    const int p = a.pos[m];
    const float2* rt = a.rope + int64_t(p) * (DH / 2);
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int d = 8 * g + 4 * fh;
      if (head < a.hq + a.hkv) {
        float rl[4], rh[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float2 cs = rt[d + e];
          const float lo = c[0][4 * g + e], hi = c[1][4 * g + e];
          rl[e] = lo * cs.x - hi * cs.y;
          rh[e] = hi * cs.x + lo * cs.y;
        }
        uint16_t* dst = (head < a.hq) ? a.q + (int64_t(m) * a.hq + head) * DH
                                      : a.kstore + a.k_off[m] + int64_t(head - a.hq) * DH;
        st_h4<DEV>(dst + d, rl[0], rl[1], rl[2], rl[3]);
        st_h4<DEV>(dst + d + DH / 2, rh[0], rh[1], rh[2], rh[3]);
      } else {
        const int gh = head - a.hq - a.hkv;
        uint16_t* dst = a.vstore + a.v_off[m];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          st_u16<DEV>(dst + int64_t(gh * DH + d + e) * a.v_stride, f2h(c[0][4 * g + e]));
          st_u16<DEV>(dst + int64_t(gh * DH + d + DH / 2 + e) * a.v_stride, f2h(c[1][4 * g + e]));
        }
      }
    }
  }
}

}  // namespace skinny
}  // namespace hs
