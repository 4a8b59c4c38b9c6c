// One block's unit of the skinny (decode-sized) fp16 MFMA GEMM.
//
// Decode re-reads every weight for a handful of rows, so the unit streams W
// rather than reusing it: a block owns a thin strip of weight rows (32, or 64
// when the epilogue needs RoPE or gate/up pairs), all M rows and one K range.
// The four waves split the range into interleaved 32-wide panels whose
// fragments they load straight into registers, several panels in flight per
// wave, so no wave waits on another until the end, where partial accumulators
// are summed through LDS and the fused epilogues run (residual add into fp32,
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
constexpr int kLdsBytes = 160 * 1024;
constexpr int kThreads = 256;
constexpr int kDeviceScope = 16;        // buffer cache-policy bit sc1: device-coherent access

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, 0x00020000);
}

// silu(z) = z / (1 + e^-z), with the hardware reciprocal (1 ulp) in place of
// an IEEE division: the result is rounded to fp16 next.
__device__ __forceinline__ float silu(float z) { return z * __builtin_amdgcn_rcpf(1.0f + __expf(-z)); }

// Weight row held in row r of strip `tile` (NR rows per strip).
//   SWIGLU: [gate 32 | up 32] for output columns 32 tile .. + 31.
//   QKV: strip s of head h (DH / 32 strips per head) holds dimensions
//     16 s .. 16 s + 15 then their rotation partners DH / 2 + 16 s .. + 15,
//     so an accumulator lane's registers 4 g + e and 4 (g + 2) + e (g < 2)
//     hold a RoPE pair.
template <int EPI, int NR, int DH>
__device__ __forceinline__ uint32_t strip_row(int tile, int r, int ffn) {
  if constexpr (EPI == EPI_SWIGLU) {
    return uint32_t((r >> 5) * ffn + tile * 32 + (r & 31));
  } else if constexpr (EPI == EPI_QKV) {
    constexpr int SPH = DH / 32;  // strips per head
    const int head = tile / SPH, sub = tile % SPH;
    return uint32_t(head * DH + (r < 16 ? 16 * sub + r : DH / 2 + 16 * sub + (r - 16)));
  } else {
    return uint32_t(tile * NR + r);
  }
}

// LDS of one block: the cross-wave reduction buffer and an arrival flag.
template <int NS, int MT>
struct SkinnyShape {
  static constexpr int RED = 4 * NS * MT * 16 * 64 * 4;
  static constexpr int SMEM = RED + 16;
};

// 32-wide K panels per chunk (a chunk is 2 (NS + MT) fragment loads).
template <int NS, int MT>
constexpr int skinny_chunk() { return NS + MT <= 3 ? 2 : 1; }

// One weight strip (`tile`) and one K split (`ks`) of a skinny GEMM, by one
// block of kThreads threads, in LDS `smem` (SkinnyShape::SMEM bytes, 1 KB
// aligned).
template <int EPI, int DH, bool W_F16, int NS, int MT>
__device__ __forceinline__ void skinny_unit(const GemmArgs& a, int tile, int ks, uint8_t* smem) {
  constexpr int NR = 32 * NS;                 // weight rows per block
  constexpr int CH = skinny_chunk<NS, MT>();
  constexpr int SMEM = SkinnyShape<NS, MT>::SMEM;
  static_assert(SMEM <= kLdsBytes, "LDS");

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
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
        pre[u] = __builtin_amdgcn_raw_buffer_load_b128(pr, row_off + uint32_t(u * 16), 0, 0);
  }
  // Operands of the epilogue that do not depend on the product, loaded now
  // so that they are in registers by then (wave w owns rows 32 w .. 32 w + 31
  // there): RESID the residual and the next norm's gains; QKV the row's
  // position, cache offsets and RoPE table entries (issued after the first
  // chunk's loads, see below).
  f32x4 res_pre[EPI == EPI_RESID ? NS : 1][4];
  f32x4 gain_pre[EPI == EPI_RESID ? NS : 1][4];
  const int m_own = wave * 32 + fr;
  const bool row_own = wave < MT && m_own < a.M;
  if constexpr (EPI == EPI_RESID) {
    if (row_own) {
#pragma unroll
      for (int i = 0; i < NS; ++i)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int n = tile * NR + i * 32 + 8 * g + 4 * fh;
          if (a.resid_f32) {
            res_pre[i][g] = *reinterpret_cast<const f32x4*>(a.resid_f32 + int64_t(m_own) * a.ldo + n);
          } else {
            float r4[4];
            load_bf16x4(a.resid + int64_t(m_own) * a.ldo + n, r4);
            res_pre[i][g] = f32x4{r4[0], r4[1], r4[2], r4[3]};
          }
          if (a.scaled_out) {
            float gm[4];
            load_bf16x4(a.gain + n, gm);
            gain_pre[i][g] = f32x4{gm[0], gm[1], gm[2], gm[3]};
          }
        }
    }
  }
  int64_t qkv_koff = 0, qkv_voff = 0;
  if constexpr (EPI == EPI_QKV) {
    if (row_own) {
      qkv_koff = a.k_off[m_own];
      qkv_voff = a.v_off[m_own];
    }
  }
  const int kt0 = ks * a.k_per_split;
  const int KT = min(a.K / BK - kt0, a.k_per_split);  // stages of this split
  const uint32_t row_bytes = uint32_t(a.K) * 2;

  const uint32_t w_rows = (EPI == EPI_SWIGLU) ? uint32_t(2 * a.ffn) : uint32_t(a.n_tiles_n * 256);
  const __amdgpu_buffer_rsrc_t wres = make_rsrc(a.W, w_rows * row_bytes);
  const __amdgpu_buffer_rsrc_t xres =
      make_rsrc(a.A, a.k8_rows ? uint32_t(a.K) * uint32_t(a.k8_rows) * 2 : uint32_t(a.M) * row_bytes);

  // Fragments go from memory straight into registers in MFMA operand layout.
  // The split's K range is cut into 32-wide panels; wave w takes panels w,
  // w + 4, w + 8, ... in chunks of CH panels and loads chunk c + 1 while it
  // multiplies chunk c.  A panel past the range is read through an empty
  // buffer resource, so it returns zeros and moves no data.
  //   weight fragment (A operand): rows strip_row(i * 32 + fr), K 16 s + 8 fh .. + 7
  //   activation fragment (B operand): rows j * 32 + fr, the same K
  static_assert(NS <= 2 && MT <= 4, "fragment slots");
  const __amdgpu_buffer_rsrc_t zres = make_rsrc(a.W, 0);
  uint32_t w_off[NS], x_off[MT];
#pragma unroll
  for (int i = 0; i < NS; ++i) {
    const uint32_t r = strip_row<EPI, NR, DH>(tile, i * 32 + fr, a.ffn);
    w_off[i] = (W_F16 ? r * 64u : r * row_bytes) + uint32_t(fh * 16);
  }
  // Activations row-major: a step is 32 bytes along the row, a panel 64.
  // k-group-major (k8_rows padded rows): a fragment is 512 contiguous bytes,
  // a step 2 k-groups and a panel 4.
  const int k8 = a.k8_rows;
#pragma unroll
  for (int j = 0; j < MT; ++j)
    x_off[j] = k8 ? uint32_t((fh * k8 + j * 32 + fr) * 16) : uint32_t(j * 32 + fr) * row_bytes + uint32_t(fh * 16);
  const uint32_t x_step = k8 ? uint32_t(2 * k8 * 16) : 32u;
  const uint32_t x_panel = k8 ? uint32_t(4 * k8 * 16) : 64u;
  const uint32_t panel_bytes = w_rows * 64;
  const int n_panels = 2 * KT;
  const int my_panels = n_panels > wave ? (n_panels - wave + 3) / 4 : 0;
  const int n_chunks = (my_panels + CH - 1) / CH;

  f32x16 acc[NS][MT];
#pragma unroll
  for (int i = 0; i < NS; ++i)
#pragma unroll
    for (int j = 0; j < MT; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  struct Chunk {
    u32x4 w[CH][2][NS];
    u32x4 x[CH][2][MT];
  };
  auto load_chunk = [&](int c, Chunk& b) {
#pragma unroll
    for (int q = 0; q < CH; ++q) {
      const int p = wave + 4 * (c * CH + q);  // panel of this split
      const bool ok = p < n_panels;
      const __amdgpu_buffer_rsrc_t wr = ok ? wres : zres;
      const __amdgpu_buffer_rsrc_t xr = ok ? xres : zres;
      const uint32_t P = uint32_t(2 * kt0 + p);  // panel of the matrix
      const uint32_t wso = W_F16 ? P * panel_bytes : P * 64u;
#pragma unroll
      for (int s = 0; s < 2; ++s) {
#pragma unroll
        for (int i = 0; i < NS; ++i)
          b.w[q][s][i] = __builtin_amdgcn_raw_buffer_load_b128(wr, w_off[i] + 32 * s, wso, 0);
#pragma unroll
        for (int j = 0; j < MT; ++j)
          b.x[q][s][j] = __builtin_amdgcn_raw_buffer_load_b128(xr, x_off[j] + x_step * s, P * x_panel, 0);
      }
    }
  };
  auto mma_chunk = [&](const Chunk& b) {
#pragma unroll
    for (int q = 0; q < CH; ++q)
#pragma unroll
      for (int s = 0; s < 2; ++s)
#pragma unroll
        for (int i = 0; i < NS; ++i) {
          const u32x4 wh = W_F16 ? b.w[q][s][i] : bf8_to_h8(b.w[q][s][i]);
#pragma unroll
          for (int j = 0; j < MT; ++j) acc[i][j] = mfma32(wh, b.x[q][s][j], acc[i][j]);
        }
  };

  // Two register sets.  Chunk 0 is always loaded (a wave without panels
  // reads zeros); later chunks are loaded only when they hold panels of this
  // wave, so the compiler's wait counts stay exact, and the scheduling
  // barriers keep each chunk's loads ahead of the previous chunk's MFMAs.
  Chunk b0, b1;
  load_chunk(0, b0);
  // QKV: the RoPE table entries of this lane's dimension pairs and, with a
  // bias, the bias of its columns (registers 4 g + e: dimension
  // 16 sub + 8 g + 4 fh + e, registers 4 (g + 2) + e: that plus DH / 2).
  float2 rope_pre[EPI == EPI_QKV ? 8 : 1];
  float bias_pre[EPI == EPI_QKV ? 16 : 1];
  if constexpr (EPI == EPI_QKV) {
    if (row_own) {
#pragma unroll
      for (int g = 0; g < 2; ++g) {
        // Pairs j .. j + 3 share one RoPE section (sections are multiples of 4 pairs).
        const int j = 16 * (tile % (DH / 32)) + 8 * g + 4 * fh;
        const float2* rt = a.rope + int64_t(rope_pos(a, m_own, j)) * (DH / 2) + j;
#pragma unroll
        for (int e = 0; e < 4; ++e) rope_pre[4 * g + e] = rt[e];
      }
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) bias_pre[r] = 0.0f;
    if (a.bias && wave < MT) {
      const uint16_t* bp = a.bias + (tile / (DH / 32)) * DH + 16 * (tile % (DH / 32)) + 4 * fh;
#pragma unroll
      for (int g = 0; g < 2; ++g) {
        load_bf16x4(bp + 8 * g, &bias_pre[4 * g]);
        load_bf16x4(bp + 8 * g + DH / 2, &bias_pre[4 * (g + 2)]);
      }
    }
  }
  __builtin_amdgcn_sched_barrier(0);
  int ch = 0;
  for (; ch + 2 < n_chunks; ch += 2) {
    load_chunk(ch + 1, b1);
    __builtin_amdgcn_sched_barrier(0);
    mma_chunk(b0);
    __builtin_amdgcn_sched_barrier(0);
    load_chunk(ch + 2, b0);
    __builtin_amdgcn_sched_barrier(0);
    mma_chunk(b1);
    __builtin_amdgcn_sched_barrier(0);
  }
  if (n_chunks - ch == 2) {
    load_chunk(ch + 1, b1);
    __builtin_amdgcn_sched_barrier(0);
    mma_chunk(b0);
    __builtin_amdgcn_sched_barrier(0);
    mma_chunk(b1);
  } else if (n_chunks - ch == 1) {
    mma_chunk(b0);
  }

  // Sum the four waves' partial accumulators through LDS ([wave][i][j][lane]
  // images of 16 floats, moved 16 bytes at a time); wave w then owns row
  // subtile j = w (MT <= 4).
  __syncthreads();
  f32x4* red = reinterpret_cast<f32x4*>(smem);
#pragma unroll
  for (int i = 0; i < NS; ++i)
#pragma unroll
    for (int j = 0; j < MT; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        red[(((wave * NS + i) * MT + j) * 64 + lane) * 4 + q] =
            f32x4{acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
  __syncthreads();
  const int j = wave;
  const bool owner = j < MT;
  f32x16 c[NS];
#pragma unroll
  for (int i = 0; i < NS; ++i)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      f32x4 v = {0.0f, 0.0f, 0.0f, 0.0f};
      if (owner) {
#pragma unroll
        for (int w = 0; w < 4; ++w) v += red[(((w * NS + i) * MT + j) * 64 + lane) * 4 + q];
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) c[i][4 * q + e] = v[e];
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
          v += res_pre[i][g];
          *reinterpret_cast<f32x4*>(orow + n) = v;
          ss += v[0] * v[0] + v[1] * v[1] + v[2] * v[2] + v[3] * v[3];
          if (a.scaled_out) {
            const f32x4 gm = gain_pre[i][g];
            store_h4(a.scaled_out + act_index(m, n, a.ldo, a.k8_rows), v[0] * gm[0], v[1] * gm[1], v[2] * gm[2],
                     v[3] * gm[3]);
          }
        }
      if (a.sumsq_out) {
        // The lane pair (fh = 0, 1) holds this row's NR columns of the strip.
        ss += __shfl_xor(ss, 32, 64);
        if (fh == 0) st_f32<false>(a.sumsq_out + int64_t(m) * strips + tile, ss);
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
    if constexpr (EPI == EPI_QKV) {
#pragma unroll
      for (int r = 0; r < 16; ++r) c[0][r] += bias_pre[r];
    }
  }
  if constexpr (EPI == EPI_SWIGLU) {
    static_assert(EPI != EPI_SWIGLU || NS == 2, "gate/up strips hold 32 + 32 rows");
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      float v[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = silu(c[0][4 * g + e]) * c[1][4 * g + e];
      store_h4(a.out + act_index(m, tile * 32 + 8 * g + 4 * fh, a.ldo, a.k8_rows), v[0], v[1], v[2], v[3]);
    }
  } else {  // EPI_QKV: a strip holds 16 dimensions of one head and their RoPE partners
    static_assert(EPI != EPI_QKV || NS == 1, "QKV strips are 32 rows");
    constexpr int SPH = DH / 32;
    const int head = tile / SPH, sub = tile % SPH;
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      const int d = 16 * sub + 8 * g + 4 * fh;  // < DH / 2; partner d + DH / 2
      if (head < a.hq + a.hkv) {
        float rl[4], rh[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float2 cs = rope_pre[4 * g + e];
          const float lo = c[0][4 * g + e], hi = c[0][4 * (g + 2) + e];
          rl[e] = lo * cs.x - hi * cs.y;
          rh[e] = hi * cs.x + lo * cs.y;
        }
        uint16_t* dst = (head < a.hq) ? a.q + (int64_t(m) * a.hq + head) * DH
                                      : a.kstore + qkv_koff + int64_t(head - a.hq) * a.kv_head_stride;
        store_h4(dst + d, rl[0], rl[1], rl[2], rl[3]);
        store_h4(dst + d + DH / 2, rh[0], rh[1], rh[2], rh[3]);
      } else {
        const int gh = head - a.hq - a.hkv;
        uint16_t* dst = a.vstore + qkv_voff + int64_t(gh) * a.kv_head_stride;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          dst[(d + e) * kv_tile_keys] = f2h(c[0][4 * g + e]);
          dst[(d + DH / 2 + e) * kv_tile_keys] = f2h(c[0][4 * (g + 2) + e]);
        }
      }
    }
  }
}

}  // namespace skinny
}  // namespace hs
