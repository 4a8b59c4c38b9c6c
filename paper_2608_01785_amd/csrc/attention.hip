// Varlen causal grouped-query flash attention for gfx950 (prefill rows).
//
// One block = 128 query rows of one sequence and one query head (4 waves x 32
// rows).  Keys/values stream through LDS in tiles of 64 keys, double
// buffered.  Scores are computed transposed, S^T = K Q^T, so each lane owns
// one query and holds 16 of its scores per 32-key subtile: the softmax row
// statistics need one cross-lane exchange (lane ^ 32) per tile.  The rows of
// K fed to the MFMA are permuted inside each 16-key block (bits 2 and 3 of
// the row index swapped), which makes the score registers line up with the
// B-operand layout of the P.V MFMA, O^T = V^T P^T, without any data movement.
// Values are stored dimension-major (V^T), so that operand is read with
// 16-byte LDS loads along the key axis.
//
// Causal alignment is bottom-right: row i of a chunk behind c cached rows
// sees keys 0 .. c + i of its own sequence only.
#include "hs_device.h"
#include "hs_kernels.h"

namespace hs {
namespace {

constexpr int BQ = 128;
constexpr int BKV = 64;
constexpr int kThreads = 256;

// MFMA row i of a 32-key subtile reads key perm32(i): bits 2 and 3 swapped.
__device__ __forceinline__ int perm32(int i) {
  return (i & ~12) | ((i >> 1) & 4) | ((i << 1) & 8);
}

// LDS swizzle of a key row: distinct for the rows perm32(0..7) read by 8 lanes.
__device__ __forceinline__ int kswz(int row) { return (row & 3) | ((row >> 1) & 4); }

template <int DH>
__global__ __launch_bounds__(kThreads, 2) void attn_kernel(AttnArgs a) {
  constexpr int KROW = DH * 2;                 // bytes per key row
  constexpr int KTILE = BKV * KROW;            // key tile bytes
  constexpr int VTILE = DH * BKV * 2;          // value tile bytes (DH rows of 128 B)
  constexpr int STAGE = KTILE + VTILE;
  constexpr int KCH = DH / 8;                  // 16-byte chunks per key row
  constexpr int KLOADS = BKV * KCH / kThreads; // per thread
  constexpr int VLOADS = DH * 8 / kThreads;
  constexpr int NDS = DH / 32;                 // output subtiles along dh
  __shared__ __attribute__((aligned(16))) uint8_t smem[2 * STAGE];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int fr = lane & 31, fh = lane >> 5;

  const int L = xcd_remap(blockIdx.x, gridDim.x);
  const int item = L / a.hq;
  const int head = L % a.hq;
  const int g = head / (a.hq / a.hkv);
  const int b = a.items[2 * item];
  const int q0 = a.items[2 * item + 1];
  const int len = a.seq_len[b];
  const int ctx = a.seq_ctx[b];
  const int row0 = a.seq_start[b];
  const int64_t kbase = a.seq_kbase[b] + int64_t(g) * DH;
  const int64_t vbase = a.seq_vbase[b] + int64_t(g) * DH * a.v_stride;
  const int kv_row_stride = a.hkv * DH;

  const int n_keys = ctx + min(q0 + BQ, len);      // keys any query of the block may see
  const int n_tiles = (n_keys + BKV - 1) / BKV;
  const int qi = min(q0 + wave * 32 + fr, len - 1);  // clamped query row (tail lanes recompute the last row)
  const int qpos = ctx + qi;
  const int wave_last = ctx + min(q0 + wave * 32 + 31, len - 1);  // last key this wave needs

  // Query fragments: B operand of S^T = K Q^T, lane = query, k = head dimension.
  u32x4 qf[DH / 16];
  {
    const uint16_t* qp = a.q + (int64_t(row0 + qi) * a.hq + head) * DH + fh * 8;
#pragma unroll
    for (int kb = 0; kb < DH / 16; ++kb) qf[kb] = *reinterpret_cast<const u32x4*>(qp + kb * 16);
  }

  u32x4 rk[KLOADS], rv[VLOADS];
  auto gload = [&](int t) {
    const int kv0 = t * BKV;
#pragma unroll
    for (int j = 0; j < KLOADS; ++j) {
      const int idx = tid + j * kThreads;
      const int row = idx / KCH, c = idx % KCH;
      rk[j] = *reinterpret_cast<const u32x4*>(a.kstore + kbase + int64_t(kv0 + row) * kv_row_stride + c * 8);
    }
#pragma unroll
    for (int j = 0; j < VLOADS; ++j) {
      const int idx = tid + j * kThreads;
      const int d = idx >> 3, c = idx & 7;
      const int key = kv0 + c * 8;
      u32x4 v = *reinterpret_cast<const u32x4*>(a.vstore + vbase + int64_t(d) * a.v_stride + key);
      if (key + 8 > n_keys) {
        // Keys past the last visible one may hold uninitialised data; P is 0
        // there, but 0 * NaN would still poison the sum, so zero them.
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t lo_ok = (key + 2 * e < n_keys) ? 0x0000ffffu : 0u;
          const uint32_t hi_ok = (key + 2 * e + 1 < n_keys) ? 0xffff0000u : 0u;
          v[e] &= (lo_ok | hi_ok);
        }
      }
      rv[j] = v;
    }
  };
  auto lstore = [&](int stage) {
    uint8_t* ks = smem + stage * STAGE;
    uint8_t* vs = ks + KTILE;
#pragma unroll
    for (int j = 0; j < KLOADS; ++j) {
      const int idx = tid + j * kThreads;
      const int row = idx / KCH, c = idx % KCH;
      const int phys = (c & ~7) | ((c & 7) ^ kswz(row));
      *reinterpret_cast<u32x4*>(ks + row * KROW + phys * 16) = rk[j];
    }
#pragma unroll
    for (int j = 0; j < VLOADS; ++j) {
      const int idx = tid + j * kThreads;
      const int d = idx >> 3, c = idx & 7;
      *reinterpret_cast<u32x4*>(vs + d * 128 + ((c ^ (d & 7)) * 16)) = rv[j];
    }
  };

  f32x16 o[NDS];
#pragma unroll
  for (int i = 0; i < NDS; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[i][r] = 0.0f;
  float m_run = -INFINITY, l_run = 0.0f;

  gload(0);
  lstore(0);
  __syncthreads();

  for (int t = 0; t < n_tiles; ++t) {
    if (t + 1 < n_tiles) gload(t + 1);
    const int kv0 = t * BKV;
    if (kv0 <= wave_last) {
      const uint8_t* ks = smem + (t & 1) * STAGE;
      const uint8_t* vs = ks + KTILE;
      f32x16 s[2];
#pragma unroll
      for (int st = 0; st < 2; ++st)
#pragma unroll
        for (int r = 0; r < 16; ++r) s[st][r] = 0.0f;
#pragma unroll
      for (int kb = 0; kb < DH / 16; ++kb) {
        const int c = 2 * kb + fh;
#pragma unroll
        for (int st = 0; st < 2; ++st) {
          const int row = 32 * st + perm32(fr);
          const int phys = (c & ~7) | ((c & 7) ^ kswz(row));
          const u32x4 kf = *reinterpret_cast<const u32x4*>(ks + row * KROW + phys * 16);
          s[st] = mfma32(kf, qf[kb], s[st]);
        }
      }
      // Register r of subtile st holds key kv0 + 32 st + 16 (r / 8) + 8 fh + r % 8.
      float mx = -INFINITY;
#pragma unroll
      for (int st = 0; st < 2; ++st)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = kv0 + 32 * st + 16 * (r >> 3) + 8 * fh + (r & 7);
          const float v = (key <= qpos) ? s[st][r] * a.scale_log2 : -INFINITY;
          s[st][r] = v;
          mx = fmaxf(mx, v);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float m_new = fmaxf(m_run, mx);
      const float alpha = exp2f(m_run - m_new);
      m_run = m_new;
      float psum = 0.0f;
#pragma unroll
      for (int st = 0; st < 2; ++st)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float p = exp2f(s[st][r] - m_new);
          s[st][r] = p;
          psum += p;
        }
      l_run = l_run * alpha + psum;
#pragma unroll
      for (int i = 0; i < NDS; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[i][r] *= alpha;
      // P^T fragments: key block kb2 (16 keys) = registers 8 (kb2 % 2) .. +8 of subtile kb2 / 2.
      u32x4 pf[4];
#pragma unroll
      for (int kb2 = 0; kb2 < 4; ++kb2) {
        const int st = kb2 >> 1, r0 = 8 * (kb2 & 1);
#pragma unroll
        for (int e = 0; e < 4; ++e) pf[kb2][e] = pack2h(s[st][r0 + 2 * e], s[st][r0 + 2 * e + 1]);
      }
#pragma unroll
      for (int i = 0; i < NDS; ++i) {
        const int d = 32 * i + fr;
#pragma unroll
        for (int kb2 = 0; kb2 < 4; ++kb2) {
          const int c = 2 * kb2 + fh;
          const u32x4 vf = *reinterpret_cast<const u32x4*>(vs + d * 128 + ((c ^ (d & 7)) * 16));
          o[i] = mfma32(vf, pf[kb2], o[i]);
        }
      }
    }
    if (t + 1 < n_tiles) lstore((t + 1) & 1);
    __syncthreads();
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  const float inv = 1.0f / l_tot;
  const int qw = q0 + wave * 32 + fr;
  if (qw < len) {
    uint16_t* op = a.o + int64_t(row0 + qw) * (a.hq * DH) + head * DH + 4 * fh;
#pragma unroll
    for (int i = 0; i < NDS; ++i)
#pragma unroll
      for (int gq = 0; gq < 4; ++gq)
        store_h4(op + 32 * i + 8 * gq, o[i][4 * gq] * inv, o[i][4 * gq + 1] * inv, o[i][4 * gq + 2] * inv,
                 o[i][4 * gq + 3] * inv);
  }
}

// ----------------------------------------------------------------------------
// Single-row attention: one block per (row, kv head, key chunk) computes the
// partial softmax statistics of all query heads of the group over its chunk;
// a second kernel merges the chunks.

template <int DH>
__global__ __launch_bounds__(kThreads, 1) void decode_attn_kernel(DecodeAttnArgs a) {
  constexpr int CK = kDecodeChunk;       // 256 keys, one per thread
  constexpr int KROW = DH * 2;
  constexpr int KCH = DH / 8;
  constexpr int VROW = CK * 2;           // 512 bytes per value row
  constexpr int VCH = CK / 8;            // 32 chunks
  constexpr int MAXG = 8;
  constexpr int PARTS = kThreads / DH;   // threads per value row in P.V
  __shared__ __attribute__((aligned(16))) uint8_t ks[CK * KROW];
  __shared__ __attribute__((aligned(16))) uint8_t vs[DH * VROW];
  __shared__ float qs[MAXG][DH];
  __shared__ float ps[MAXG][CK];
  __shared__ float red[4][MAXG];
  __shared__ float ored[PARTS][MAXG][DH];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int4 it = a.items[blockIdx.x];
  const int r = it.x, g = it.y, c = it.z;
  const int4 rw = a.rows[r];
  const int t = rw.x, b = rw.y;
  const int G = a.hq / a.hkv;
  const int n_keys = a.seq_ctx[b] + 1;
  const int k0 = c * CK;
  const int nk = min(CK, n_keys - k0);
  const int64_t kbase = a.seq_kbase[b] + int64_t(g) * DH + int64_t(k0) * a.hkv * DH;
  const int64_t vbase = a.seq_vbase[b] + int64_t(g) * DH * a.v_stride + k0;

  for (int i = tid; i < G * DH; i += kThreads) {
    const int hh = i / DH, d = i % DH;
    qs[hh][d] = h2f(a.q[(int64_t(t) * a.hq + g * G + hh) * DH + d]);
  }
  for (int i = tid; i < CK * KCH; i += kThreads) {
    const int row = i / KCH, cc = i % KCH;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (row < nk) v = *reinterpret_cast<const u32x4*>(a.kstore + kbase + int64_t(row) * a.hkv * DH + cc * 8);
    const int phys = (cc & ~7) | ((cc & 7) ^ (row & 7));
    *reinterpret_cast<u32x4*>(ks + row * KROW + phys * 16) = v;
  }
  for (int i = tid; i < DH * VCH; i += kThreads) {
    const int d = i / VCH, cc = i % VCH;
    const int key = cc * 8;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (key < nk) {
      v = *reinterpret_cast<const u32x4*>(a.vstore + vbase + int64_t(d) * a.v_stride + key);
      if (key + 8 > nk) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t lo_ok = (key + 2 * e < nk) ? 0x0000ffffu : 0u;
          const uint32_t hi_ok = (key + 2 * e + 1 < nk) ? 0xffff0000u : 0u;
          v[e] &= (lo_ok | hi_ok);
        }
      }
    }
    const int phys = (cc & ~7) | ((cc & 7) ^ (d & 7));
    *reinterpret_cast<u32x4*>(vs + d * VROW + phys * 16) = v;
  }
  __syncthreads();

  // Scores: thread j owns key k0 + j.
  float sc[MAXG];
  {
    const int j = tid;
#pragma unroll
    for (int hh = 0; hh < MAXG; ++hh) sc[hh] = 0.0f;
#pragma unroll
    for (int cc = 0; cc < KCH; ++cc) {
      const int phys = (cc & ~7) | ((cc & 7) ^ (j & 7));
      const u32x4 kv = *reinterpret_cast<const u32x4*>(ks + j * KROW + phys * 16);
      float kf[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) h2x_to_f(kv[e], kf[2 * e], kf[2 * e + 1]);
#pragma unroll
      for (int hh = 0; hh < MAXG; ++hh) {
        if (hh < G) {
#pragma unroll
          for (int e = 0; e < 8; ++e) sc[hh] += qs[hh][cc * 8 + e] * kf[e];
        }
      }
    }
#pragma unroll
    for (int hh = 0; hh < MAXG; ++hh) sc[hh] = (j < nk) ? sc[hh] * a.scale_log2 : -INFINITY;
  }
  float mh[MAXG], lh[MAXG];
#pragma unroll
  for (int hh = 0; hh < MAXG; ++hh) {
    if (hh < G) {
      const float m = wave_max(sc[hh]);
      if (lane == 0) red[wave][hh] = m;
    }
  }
  __syncthreads();
#pragma unroll
  for (int hh = 0; hh < MAXG; ++hh) {
    if (hh < G) {
      mh[hh] = fmaxf(fmaxf(red[0][hh], red[1][hh]), fmaxf(red[2][hh], red[3][hh]));
      const float p = exp2f(sc[hh] - mh[hh]);
      ps[hh][tid] = p;
      sc[hh] = p;
    }
  }
  __syncthreads();
#pragma unroll
  for (int hh = 0; hh < MAXG; ++hh) {
    if (hh < G) {
      const float s = wave_sum(sc[hh]);
      if (lane == 0) red[wave][hh] = s;
    }
  }
  __syncthreads();
#pragma unroll
  for (int hh = 0; hh < MAXG; ++hh)
    if (hh < G) lh[hh] = red[0][hh] + red[1][hh] + red[2][hh] + red[3][hh];

  // P.V: thread -> (value row d, key part).
  {
    const int d = tid % DH, part = tid / DH;
    constexpr int KPP = CK / PARTS;  // keys per part
    float acc[MAXG];
#pragma unroll
    for (int hh = 0; hh < MAXG; ++hh) acc[hh] = 0.0f;
#pragma unroll 4
    for (int cc = part * (KPP / 8); cc < (part + 1) * (KPP / 8); ++cc) {
      const int phys = (cc & ~7) | ((cc & 7) ^ (d & 7));
      const u32x4 vv = *reinterpret_cast<const u32x4*>(vs + d * VROW + phys * 16);
      float vf[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) h2x_to_f(vv[e], vf[2 * e], vf[2 * e + 1]);
#pragma unroll
      for (int hh = 0; hh < MAXG; ++hh)
        if (hh < G) {
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[hh] += ps[hh][cc * 8 + e] * vf[e];
        }
    }
#pragma unroll
    for (int hh = 0; hh < MAXG; ++hh)
      if (hh < G) ored[part][hh][d] = acc[hh];
  }
  __syncthreads();
  for (int i = tid; i < G * DH; i += kThreads) {
    const int hh = i / DH, d = i % DH;
    float s = 0.0f;
#pragma unroll
    for (int p = 0; p < PARTS; ++p) s += ored[p][hh][d];
    a.part_o[(int64_t(blockIdx.x) * G + hh) * DH + d] = s;
  }
  if (tid < G) {
    // mh/lh are identical in every thread; thread hh publishes head hh.
    float m = 0.0f, l = 0.0f;
#pragma unroll
    for (int hh = 0; hh < MAXG; ++hh)
      if (hh == tid) { m = mh[hh]; l = lh[hh]; }
    a.part_ml[(int64_t(blockIdx.x) * G + tid) * 2 + 0] = m;
    a.part_ml[(int64_t(blockIdx.x) * G + tid) * 2 + 1] = l;
  }
}

template <int DH>
__global__ __launch_bounds__(128) void decode_combine_kernel(DecodeAttnArgs a) {
  const int r = blockIdx.x / a.hq;
  const int h = blockIdx.x % a.hq;
  const int G = a.hq / a.hkv;
  const int g = h / G, hh = h % G;
  const int4 rw = a.rows[r];
  const int t = rw.x, first = rw.z, nch = rw.w;
  const int d = threadIdx.x;
  if (d >= DH) return;
  float m = -INFINITY;
  for (int c = 0; c < nch; ++c) {
    const int64_t item = first + int64_t(g) * nch + c;
    m = fmaxf(m, a.part_ml[(item * G + hh) * 2]);
  }
  float num = 0.0f, den = 0.0f;
  for (int c = 0; c < nch; ++c) {
    const int64_t item = first + int64_t(g) * nch + c;
    const float w = exp2f(a.part_ml[(item * G + hh) * 2] - m);
    den += w * a.part_ml[(item * G + hh) * 2 + 1];
    num += w * a.part_o[(item * G + hh) * DH + d];
  }
  a.o[int64_t(t) * a.hq * DH + h * DH + d] = f2h(num / den);
}

}  // namespace

hipError_t launch_attention(const AttnArgs& a, hipStream_t s) {
  if (a.n_items <= 0) return hipSuccess;
  const int grid = a.n_items * a.hq;
  if (a.dh == 64)
    hipLaunchKernelGGL(attn_kernel<64>, dim3(grid), dim3(kThreads), 0, s, a);
  else
    hipLaunchKernelGGL(attn_kernel<128>, dim3(grid), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_decode_attention(const DecodeAttnArgs& a, hipStream_t s) {
  if (a.n_items <= 0) return hipSuccess;
  if (a.dh == 64) {
    hipLaunchKernelGGL(decode_attn_kernel<64>, dim3(a.n_items), dim3(kThreads), 0, s, a);
    hipLaunchKernelGGL(decode_combine_kernel<64>, dim3(a.n_rows * a.hq), dim3(64), 0, s, a);
  } else {
    hipLaunchKernelGGL(decode_attn_kernel<128>, dim3(a.n_items), dim3(kThreads), 0, s, a);
    hipLaunchKernelGGL(decode_combine_kernel<128>, dim3(a.n_rows * a.hq), dim3(128), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace hs
