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
#include "decode_unit.h"

namespace hs {
namespace {

constexpr int BQ = 128;
constexpr int BKV = 64;
constexpr int kThreads = 256;

// LDS placement of 16-byte chunk c of key row r (DH * 2 bytes per row).  A
// 16-lane pass of fragment reads takes one logical chunk of 16 distinct rows
// (perm32 of 16 consecutive indices).  With 256-byte rows every row starts on
// bank 0, so the 16 rows need 16 different physical chunks (c ^ (r & 15));
// with 128-byte rows odd rows start on bank 32, so the chunks need only
// differ within each parity (c ^ ((r >> 1) & 7)).
template <int DH>
__device__ __forceinline__ int kphys(int r, int c) {
  return DH == 128 ? (c ^ (r & 15)) : (c ^ ((r >> 1) & 7));
}

// Chunk c (8 keys) of value row d (64 keys, 128 bytes): odd rows start on bank
// 32, so a pass over 16 consecutive rows needs distinct chunks per parity.
__device__ __forceinline__ int vphys(int d, int c) { return c ^ ((d >> 1) & 7); }

// Buffer resource over the cache array `base` from element `off` on: the
// 64-bit start is block-uniform, so it is moved to scalar registers; tile
// loads then take a per-lane constant offset plus a uniform tile offset and
// need no vector address arithmetic.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t cache_rsrc(const uint16_t* base, int64_t off) {
  const uint64_t addr = reinterpret_cast<uint64_t>(base + off);
  const uint32_t lo = __builtin_amdgcn_readfirstlane(uint32_t(addr));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(uint32_t(addr >> 32));
  return __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<void*>((uint64_t(hi) << 32) | lo), 0, 0x7ffffff0,
                                           0x00020000);
}

// Two fp32 values -> two fp16 values (round to nearest even), one instruction.
__device__ __forceinline__ uint32_t pack2h_rne(float lo, float hi) {
  typedef float f2 __attribute__((ext_vector_type(2)));
  typedef _Float16 h2 __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f2{lo, hi}), h2));
}

// The reference maximum of the online softmax moves only when a tile's
// maximum exceeds it by more than this (log2 units): weights are then at
// most 2^8, well inside fp16, and the output rescale is skipped on almost
// every tile.  Any reference value gives the same softmax; only rounding
// differs.
constexpr float kLazyMax = 8.0f;

// One online-softmax step over a 64-key tile of scores held as two 32-key
// subtiles (register r of subtile st: key kv0 + 32 st + 16 (r / 8) + 8 fh +
// r % 8 of the lane's query).  `lim` = qpos - kv0 - 8 fh: keys with
// 32 st + 16 (r / 8) + r % 8 > lim are masked when `mask` is set.  The
// weights are left in `pf` as the B operand of O^T = V^T P^T.
template <int NDS>
__device__ __forceinline__ void softmax_tile(f32x16 (&s)[2], f32x16 (&o)[NDS], u32x4 (&pf)[4], float& m_run,
                                             float& l_run, float scale_log2, bool mask, int lim) {
  if (mask) {
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (32 * st + 16 * (r >> 3) + (r & 7) > lim) s[st][r] = -INFINITY;
  }
  float mx = -INFINITY;
#pragma unroll
  for (int st = 0; st < 2; ++st)
#pragma unroll
    for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[st][r]);
  mx = fmaxf(mx, __shfl_xor(mx, 32, 64)) * scale_log2;
  // A row that has seen no key yet keeps -inf; its exponents are taken
  // against 0, which gives weight 0.
  const bool move = mx > m_run + kLazyMax;
  const float m_new = move ? mx : m_run;
  const float m_use = m_new == -INFINITY ? 0.0f : m_new;
  const float alpha = exp2_raw(m_run - m_use);
  m_run = m_new;
  float psum = 0.0f;
#pragma unroll
  for (int st = 0; st < 2; ++st)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const float p = exp2_raw(fmaf(s[st][r], scale_log2, -m_use));
      s[st][r] = p;
      psum += p;
    }
  l_run = l_run * alpha + psum;
  if (__ballot(move) != 0) {
#pragma unroll
    for (int i = 0; i < NDS; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[i][r] *= alpha;
  }
  // P^T fragments: key block kb2 (16 keys) = registers 8 (kb2 % 2) .. +8 of subtile kb2 / 2.
#pragma unroll
  for (int kb2 = 0; kb2 < 4; ++kb2) {
    const int st = kb2 >> 1, r0 = 8 * (kb2 & 1);
#pragma unroll
    for (int e = 0; e < 4; ++e) pf[kb2][e] = pack2h_rne(s[st][r0 + 2 * e], s[st][r0 + 2 * e + 1]);
  }
}

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
  LaunchClock clk;
  clk.begin(a.clock);

  // Units L = item * hq + head are ordered longest key range first, and the
  // Gq = hq / hkv consecutive units of a group share one key/value head.
  // Work-groups go to the XCDs round-robin (block b to XCD b % 8), so XCD x
  // takes groups x, x + 8, x + 16, ... in order: every XCD gets an equal share
  // of the longest-first list, and a group's units run on one XCD, where its
  // keys and values stay in that XCD's L2.  The grid is padded to whole rounds
  // of groups; padding blocks exit.
  const int Gq = a.hq / a.hkv;
  const int xcd = blockIdx.x % kNumXcd, kx = blockIdx.x / kNumXcd;
  const int L = ((kx / Gq) * kNumXcd + xcd) * Gq + kx % Gq;
  if (L >= a.n_items * a.hq) return;
  const int item = L / a.hq;
  const int head = L % a.hq;
  const int g = head / (a.hq / a.hkv);
  const int b = a.items[2 * item];
  const int q0 = a.items[2 * item + 1];
  const int len = a.seq_len[b];
  const int ctx = a.seq_ctx[b];
  const int row0 = a.seq_start[b];
  const int64_t* pages = a.page_base + a.seq_page0[b];
  const int64_t head_off = int64_t(g) * a.kv_head_stride;

  // Causal: row i sees keys 0 .. ctx + i.  Bidirectional: every row sees all
  // ctx + len keys, which is the causal rule applied as if every row sat at
  // the sequence's last position.
  const bool bidir = a.bidirectional != 0;
  const int n_keys = ctx + (bidir ? len : min(q0 + BQ, len));  // keys any query of the block may see
  const int n_tiles = (n_keys + BKV - 1) / BKV;
  const int qi = min(q0 + wave * 32 + fr, len - 1);  // clamped query row (tail lanes recompute the last row)
  const int qpos = bidir ? ctx + len - 1 : ctx + qi;
  const int wave_last = bidir ? ctx + len - 1 : ctx + min(q0 + wave * 32 + 31, len - 1);  // last key needed
  const int wave_first = bidir ? ctx + len - 1 : ctx + min(q0 + wave * 32, len - 1);  // first row's position

  // Query fragments: B operand of S^T = K Q^T, lane = query, k = head dimension.
  u32x4 qf[DH / 16];
  {
    const uint16_t* qp = a.q + (int64_t(row0 + qi) * a.hq + head) * DH + fh * 8;
#pragma unroll
    for (int kb = 0; kb < DH / 16; ++kb) qf[kb] = *reinterpret_cast<const u32x4*>(qp + kb * 16);
  }

  // Per-lane byte offsets of the tile loads inside a page; a tile adds the
  // uniform offset of its first key.  A value tile of 64 keys is two
  // consecutive 32-key value tiles of the cache.
  uint32_t koff[KLOADS], voff[VLOADS];
#pragma unroll
  for (int j = 0; j < KLOADS; ++j) {
    const int idx = tid + j * kThreads;
    koff[j] = uint32_t(((idx / KCH) * DH + (idx % KCH) * 8) * 2);
  }
#pragma unroll
  for (int j = 0; j < VLOADS; ++j) {
    const int idx = tid + j * kThreads;
    const int d = idx >> 3, c = idx & 7;
    voff[j] = uint32_t(((c >> 2) * kv_tile_keys * DH + d * kv_tile_keys + (c & 3) * 8) * 2);
  }
  u32x4 rk[KLOADS], rv[VLOADS];
  // pg: page-table entry of the tile the next gload fetches, read one tile
  // ahead (index clamped, so the read is unconditional and in bounds).
  const int t_end = n_tiles - 1;
  auto gload = [&](int t, int64_t pg) {
    const int kv0 = t * BKV;
    const uint32_t so = uint32_t((kv0 % a.page_keys) * DH * 2);
    const __amdgpu_buffer_rsrc_t kres = cache_rsrc(a.kstore, pg + head_off);
    const __amdgpu_buffer_rsrc_t vres = cache_rsrc(a.vstore, pg + head_off);
#pragma unroll
    for (int j = 0; j < KLOADS; ++j) rk[j] = __builtin_amdgcn_raw_buffer_load_b128(kres, koff[j], so, 0);
#pragma unroll
    for (int j = 0; j < VLOADS; ++j) rv[j] = __builtin_amdgcn_raw_buffer_load_b128(vres, voff[j], so, 0);
  };
  // Values of keys past the last visible one may be uninitialised; their
  // weights are 0, but 0 * NaN would still poison the sum, so the last tile's
  // are zeroed before they reach LDS.
  auto vmask = [&](int t) {
    if (t * BKV + BKV <= n_keys) return;
#pragma unroll
    for (int j = 0; j < VLOADS; ++j) {
      const int key = t * BKV + ((tid + j * kThreads) & 7) * 8;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t lo_ok = (key + 2 * e < n_keys) ? 0x0000ffffu : 0u;
        const uint32_t hi_ok = (key + 2 * e + 1 < n_keys) ? 0xffff0000u : 0u;
        rv[j][e] &= (lo_ok | hi_ok);
      }
    }
  };
  auto lstore = [&](int stage) {
    uint8_t* ks = smem + stage * STAGE;
    uint8_t* vs = ks + KTILE;
#pragma unroll
    for (int j = 0; j < KLOADS; ++j) {
      const int idx = tid + j * kThreads;
      const int row = idx / KCH, c = idx % KCH;
      const int phys = kphys<DH>(row, c);
      *reinterpret_cast<u32x4*>(ks + row * KROW + phys * 16) = rk[j];
    }
#pragma unroll
    for (int j = 0; j < VLOADS; ++j) {
      const int idx = tid + j * kThreads;
      const int d = idx >> 3, c = idx & 7;
      *reinterpret_cast<u32x4*>(vs + d * 128 + vphys(d, c) * 16) = rv[j];
    }
  };

  f32x16 o[NDS];
#pragma unroll
  for (int i = 0; i < NDS; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[i][r] = 0.0f;
  float m_run = -INFINITY, l_run = 0.0f;

  gload(0, pages[0]);
  vmask(0);
  lstore(0);
  int64_t pg = pages[min(1, t_end) * BKV / a.page_keys];
  __syncthreads();

  for (int t = 0; t < n_tiles; ++t) {
    if (t + 1 < n_tiles) gload(t + 1, pg);
    pg = pages[min(t + 2, t_end) * BKV / a.page_keys];
    const int kv0 = t * BKV;
    if (kv0 <= wave_last) {
      const uint8_t* ks = smem + (t & 1) * STAGE;
      const uint8_t* vs = ks + KTILE;
      f32x16 s[2];
#pragma unroll
      for (int st = 0; st < 2; ++st)
#pragma unroll
        for (int r = 0; r < 16; ++r) s[st][r] = 0.0f;
      // K fragments are read one 16-wide step ahead of the MFMAs that use
      // them (two independent accumulator chains, one per 32-key half), so
      // each MFMA waits for a read issued a step earlier, not for its own.
      auto kfrag = [&](int kb, int st) {
        const int row = 32 * st + perm32(fr);
        return *reinterpret_cast<const u32x4*>(ks + row * KROW + kphys<DH>(row, 2 * kb + fh) * 16);
      };
      u32x4 kf[2][2];
      kf[0][0] = kfrag(0, 0);
      kf[0][1] = kfrag(0, 1);
    __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // the first step's reads lead the pipeline
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // the first step's reads lead the pipeline
#pragma unroll
      for (int kb = 0; kb < DH / 16; ++kb) {
        if (kb + 1 < DH / 16) {
          kf[(kb + 1) & 1][0] = kfrag(kb + 1, 0);
          kf[(kb + 1) & 1][1] = kfrag(kb + 1, 1);
        }
        s[0] = mfma32(kf[kb & 1][0], qf[kb], s[0]);
        s[1] = mfma32(kf[kb & 1][1], qf[kb], s[1]);
        if (kb + 1 < DH / 16) {
          __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // the next step's two reads
          __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);  // then this step's two MFMAs
        }
      }
      __builtin_amdgcn_sched_barrier(0);
      // Only tiles reaching past the wave's first query position need the
      // causal mask (every key of an earlier tile is visible to all of the
      // wave's rows and lies inside the sequence).  The maximum is taken on
      // the raw scores (the scale is positive) and the scale is folded into
      // the exponent's FMA; masked scores are -inf and give 0.
      u32x4 pf[4];
      softmax_tile<NDS>(s, o, pf, m_run, l_run, a.scale_log2, kv0 + BKV - 1 > wave_first, qpos - kv0 - 8 * fh);
      // V fragments likewise one 16-key step ahead; the NDS output subtiles
      // are independent accumulator chains.
      auto vfrag = [&](int kb2, int i) {
        const int d = 32 * i + fr;
        return *reinterpret_cast<const u32x4*>(vs + d * 128 + vphys(d, 2 * kb2 + fh) * 16);
      };
      u32x4 vf[2][NDS];
#pragma unroll
      for (int i = 0; i < NDS; ++i) vf[0][i] = vfrag(0, i);
    __builtin_amdgcn_sched_group_barrier(0x100, NDS, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, NDS, 0);
#pragma unroll
      for (int kb2 = 0; kb2 < 4; ++kb2) {
        if (kb2 + 1 < 4) {
#pragma unroll
          for (int i = 0; i < NDS; ++i) vf[(kb2 + 1) & 1][i] = vfrag(kb2 + 1, i);
        }
#pragma unroll
        for (int i = 0; i < NDS; ++i) o[i] = mfma32(vf[kb2 & 1][i], pf[kb2], o[i]);
        if (kb2 + 1 < 4) {
          __builtin_amdgcn_sched_group_barrier(0x100, NDS, 0);  // the next step's reads
          __builtin_amdgcn_sched_group_barrier(0x008, NDS, 0);  // then this step's MFMAs
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    if (t + 1 < n_tiles) {
      vmask(t + 1);
      lstore((t + 1) & 1);
    }
    __syncthreads();
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  const float inv = 1.0f / l_tot;
  const int qw = q0 + wave * 32 + fr;
  if (qw < len) {
    // Groups 2p and 2p + 1 of a subtile leave as one 16-byte store per lane:
    // eight consecutive dimensions, one k-group of the row in either layout.
#pragma unroll
    for (int i = 0; i < NDS; ++i)
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        float lo[4], hi[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          lo[e] = o[i][8 * p + e] * inv;
          hi[e] = o[i][8 * p + 4 + e] * inv;
        }
        const u32x4 v = swap_h8(lo, hi);
        *reinterpret_cast<u32x4*>(a.o + act_index(row0 + qw, head * DH + 32 * i + 16 * p + 8 * fh, a.hq * DH,
                                                  a.o_k8_rows)) = v;
      }
  }
  clk.end(a.clock);
}

// ----------------------------------------------------------------------------
// Single-row (decode) attention: one block per (work item, key/value head);
// the unit is in decode_unit.h.
template <int DH>
__global__ __launch_bounds__(kThreads, 2) void decode_attn_kernel(DecodeAttnArgs a) {
  __shared__ decode::DecodeSmem<DH> sm;
  const int item = blockIdx.x / a.hkv;
  if (a.n_items_dev && item >= *a.n_items_dev) return;  // a grid sized for a fixed layout
  decode::decode_attn_unit<DH>(a, item, blockIdx.x % a.hkv, sm);
}

}  // namespace

hipError_t launch_attention(const AttnArgs& a, hipStream_t s) {
  if (a.n_items <= 0) return hipSuccess;
  // Whole rounds of key/value-head groups over the XCDs (see attn_kernel).
  const int groups = a.n_items * a.hkv;
  const int grid = (groups + kNumXcd - 1) / kNumXcd * kNumXcd * (a.hq / a.hkv);
  if (a.dh == 64)
    hipLaunchKernelGGL(attn_kernel<64>, dim3(grid), dim3(kThreads), 0, s, a);
  else
    hipLaunchKernelGGL(attn_kernel<128>, dim3(grid), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_decode_attention(const DecodeAttnArgs& a, hipStream_t s) {
  if (a.n_items <= 0) return hipSuccess;
  const int grid = a.n_items * a.hkv;
  if (a.dh == 64)
    hipLaunchKernelGGL(decode_attn_kernel<64>, dim3(grid), dim3(kThreads), 0, s, a);
  else
    hipLaunchKernelGGL(decode_attn_kernel<128>, dim3(grid), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace hs
