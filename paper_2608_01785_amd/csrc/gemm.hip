// Persistent fp16 MFMA GEMM for gfx950 with fused epilogues.
//
// Computes C[M, N] = A[M, K] * W[N, K]^T (fp16 activations times [out, in]
// weights, fp32 accumulation).  Weights are either bf16 row-major, converted
// to fp16 after they leave LDS (exact for the weight range), or prepared fp16
// in panel-major order [K / 32][N][32], which makes every stage of a tile one
// contiguous run.  Both MFMA operands are fp16: the same MFMA rate as bf16 on
// gfx950 with 8x finer rounding of the activations.
//
// The MFMA is issued as C^T = W * A^T: the weight tile is the MFMA A operand
// and the activation tile the B operand, so every lane of the 32x32
// accumulator owns one activation row and four consecutive output columns per
// register group.  That makes 8-byte output stores possible and keeps the
// pairs the epilogues need (RoPE's (j, j + dh/2), SwiGLU's gate/up) in the
// same lane and register.
//
// Block tile 256 (weight rows) x 256 (activation rows), 4 waves in a 2 x 2
// grid, each wave 128 x 128 = 4 x 4 MFMA tiles of 32x32x16.  K advances in
// slabs of 32 through a ring of 4 LDS stages (128 KB): both operands are
// copied buffer -> LDS by the load unit itself (no staging registers), so
// three slabs are in flight while the fourth feeds the MFMAs.  A five-stage
// ring measured about 5 % slower on the large shapes and a three-stage one
// the same as four (plausibly because 32 CUs x 5 x 32 KB in flight exceeds
// the XCD's 4 MB L2, which neighbouring blocks share).
// The grid is persistent (one block per CU of the budget); blocks walk the
// tile space in grouped order, remapped so each XCD takes a contiguous range.
#include <type_traits>

#include "hs_device.h"
#include "hs_kernels.h"

namespace hs {
namespace {

constexpr int BM = 256;   // activation rows per tile
constexpr int BN = 256;   // weight rows per tile
constexpr int BK = 32;    // K per LDS stage
constexpr int kStages = 4;
constexpr int kThreads = 256;
constexpr int kRowBytes = BK * 2;            // 64 bytes = 4 chunks of 16
constexpr int kTileBytes = 256 * kRowBytes;  // 16 KB
constexpr int kStageBytes = 2 * kTileBytes;  // weight tile + activation tile
constexpr int kGroupM = 4;

// Row of W that lands in tile row r (0..255) of output tile tile_n.
template <int EPI>
__device__ __forceinline__ uint32_t weight_row(int tile_n, int r, int ffn) {
  if constexpr (EPI == EPI_SWIGLU) {
    // Tile rows: [wave-n 0: gate 64 | up 64][wave-n 1: gate 64 | up 64] for
    // output columns tile_n * 128 .. +128.
    const int half = r >> 7, rr = r & 127, up = rr >> 6, jj = rr & 63;
    return uint32_t(up * ffn + tile_n * 128 + half * 64 + jj);
  } else {
    return uint32_t(tile_n * BN + r);
  }
}

// 16-byte chunk c of tile row r sits at physical chunk c ^ swz(r): the 8 rows
// read by 8 consecutive lanes then cover all 32 banks.
__device__ __forceinline__ int swz(int r) { return (r >> 1) & 3; }

__device__ __forceinline__ float silu(float z) { return z / (1.0f + __expf(-z)); }

using lds_ptr_t = __attribute__((address_space(3))) void*;

// Buffer resource over [base, base + bytes): loads past the end return zero.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, 0x00020000);
}

// Workgroup barrier without the compiler's memory fence (which would wait for
// every outstanding copy).  Callers wait for exactly the copies they need
// first; LDS reads of the previous stage have completed because their results
// were consumed.
__device__ __forceinline__ void barrier_nofence() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Wait until at most n vector-memory operations of this wave are outstanding.
__device__ __forceinline__ void wait_vm(int n) {
  switch (n) {
    case 0: asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); break;
    case 1: asm volatile("s_waitcnt vmcnt(8)" ::: "memory"); break;
    case 2: asm volatile("s_waitcnt vmcnt(16)" ::: "memory"); break;
    default: asm volatile("s_waitcnt vmcnt(24)" ::: "memory"); break;
  }
}

template <int EPI, int DH, bool W_F16>
__global__ __launch_bounds__(kThreads, 1) void gemm_kernel(GemmArgs a) {
  __shared__ __attribute__((aligned(1024))) uint8_t smem[kStages * kStageBytes];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wn = wave & 1;   // weight-row half of the tile
  const int wm = wave >> 1;  // activation-row half of the tile
  const int fr = lane & 31;
  const int fh = lane >> 5;

  const int n_m_tiles = (a.M + BM - 1) / BM;
  const int n_tiles = n_m_tiles * a.n_tiles_n;
  const int KT = a.K / BK;
  const uint32_t row_bytes = uint32_t(a.K) * 2;
  const uint32_t w_rows = (EPI == EPI_SWIGLU) ? uint32_t(2 * a.ffn) : uint32_t(a.n_tiles_n * BN);
  const __amdgpu_buffer_rsrc_t wres = make_rsrc(a.W, w_rows * row_bytes);
  const __amdgpu_buffer_rsrc_t ares = make_rsrc(a.A, uint32_t(a.M) * row_bytes);

  // Loads: one wave instruction fills 16 consecutive tile rows (1 KB); lane i
  // lands at byte 16 i = row i / 4, physical chunk i % 4, so it fetches logical
  // chunk (i % 4) ^ swz(row).  Wave w fills rows 64 w .. 64 w + 63 of both tiles.
  const int ld_sub = lane >> 2;
  const int ld_chunk = (lane & 3) ^ swz(ld_sub);  // rows 16 j + ld_sub share swz with ld_sub

  const int per_group = kGroupM * a.n_tiles_n;
  auto tile_coords = [&](int L, int& tile_m, int& tile_n) {
    const int group = L / per_group;
    const int first_m = group * kGroupM;
    const int gsize = min(n_m_tiles - first_m, kGroupM);
    tile_m = first_m + (L % per_group) % gsize;
    tile_n = (L % per_group) / gsize;
  };

  uint32_t w_off[4], a_off[4];
  // fp16 weights are panel-major ([K / 32][N][32]): one stage of a weight row
  // is 64 contiguous bytes and a tile's stage one contiguous 16 KB run.
  const uint32_t w_row_stride = W_F16 ? uint32_t(kRowBytes) : row_bytes;
  const uint32_t w_stage_stride = W_F16 ? w_rows * kRowBytes : uint32_t(kRowBytes);
  // A half unit (hm = 0 or 1) covers activation rows hm * 128 .. + 127 of its
  // tile: LDS activation rows 0..127 hold them (copied by waves 0 and 1);
  // waves 2 and 3 copy the same rows again into the unused rows 128..255, so
  // every stage still has exactly 8 copies per wave for the vmcnt accounting.
  auto set_tile = [&](int tile_m, int tile_n, int hm) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = wave * 64 + 16 * j + ld_sub;
      const int ar = hm < 0 ? r : hm * 128 + (r & 127);
      w_off[j] = weight_row<EPI>(tile_n, r, a.ffn) * w_row_stride + ld_chunk * 16;
      a_off[j] = uint32_t(tile_m * BM + ar) * row_bytes + ld_chunk * 16;  // rows >= M read zero
    }
  };
  auto issue_stage = [&](int kt, int buf) {
    const int koff = kt * BK * 2;
    const uint32_t wkoff = uint32_t(kt) * w_stage_stride;
    uint8_t* wbase = smem + buf * kStageBytes + wave * 64 * kRowBytes;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(wres, (lds_ptr_t)(wbase + j * 16 * kRowBytes), 16, w_off[j], wkoff,
                                               0, 0);
#pragma unroll
    for (int j = 0; j < 4; ++j)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ares, (lds_ptr_t)(wbase + kTileBytes + j * 16 * kRowBytes), 16,
                                               a_off[j], koff, 0, 0);
  };

  // Fragments of one half stage (16-wide K step kk): [i] weight, [j] activation.
  // JT = activation subtiles per wave: 4 (full tile, rows wm * 128 ..) or 2
  // (half unit, rows wm * 64 ..).
  struct Half {
    u32x4 w[4], a[4];
  };
  auto read_half = [&](auto jt, int buf, int kk, Half& h) {
    constexpr int JT = decltype(jt)::value;
    const uint8_t* base = smem + buf * kStageBytes;
    const int phys = (kk * 2 + fh) ^ swz(fr);
#pragma unroll
    for (int i = 0; i < 4; ++i)
      h.w[i] = *reinterpret_cast<const u32x4*>(base + (wn * 128 + i * 32 + fr) * kRowBytes + phys * 16);
#pragma unroll
    for (int j = 0; j < JT; ++j)
      h.a[j] = *reinterpret_cast<const u32x4*>(base + kTileBytes + (wm * JT * 32 + j * 32 + fr) * kRowBytes +
                                               phys * 16);
  };

  // Work units: full tiles, except that when the last round would leave more
  // than half the blocks idle its tiles are split into two 128-row halves.
  // Each output element is accumulated in the same order either way, so the
  // result does not depend on the grid.
  const int G = gridDim.x;
  const int full_units = (n_tiles / G) * G;
  const int tail = n_tiles - full_units;
  const bool split_tail = tail > 0 && 2 * tail <= G;
  const int n_units = split_tail ? full_units + 2 * tail : n_tiles;
  auto unit_coords = [&](int u, int& tile_m, int& tile_n, int& hm) {
    int t = u;
    hm = -1;
    if (split_tail && u >= full_units) {
      t = full_units + (u - full_units) / 2;
      hm = (u - full_units) % 2;
    }
    tile_coords(t, tile_m, tile_n);
  };

  int L = xcd_remap(blockIdx.x, G);
  if (L >= n_units) return;
  int tile_m, tile_n, hm;
  unit_coords(L, tile_m, tile_n, hm);
  set_tile(tile_m, tile_n, hm);
#pragma unroll
  for (int st = 0; st < kStages - 1; ++st)
    if (st < KT) issue_stage(st, st);

  f32x16 acc[4][4];
  while (true) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    auto mfma_half = [&](auto jt, const Half& h) {
      constexpr int JT = decltype(jt)::value;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const u32x4 wh = W_F16 ? h.w[i] : bf8_to_h8(h.w[i]);
#pragma unroll
        for (int j = 0; j < JT; ++j) acc[i][j] = mfma32(wh, h.a[j], acc[i][j]);
      }
    };

    // Stage s lives in buffer s % kStages.  Each 16-wide half of a stage is
    // read from LDS while the previous half multiplies, so LDS reads are
    // spread over the MFMA stream instead of bursting after the barrier.  The
    // barrier of stage s sits between its two halves: by then every wave has
    // read all of stage s, so its buffer can be refilled.
    auto k_loop = [&](auto jt) {
      constexpr int JT = decltype(jt)::value;
      constexpr int NM = 4 * JT;  // MFMAs per half stage
      wait_vm(min(kStages - 2, KT - 1));
      barrier_nofence();
      if (kStages - 1 < KT) issue_stage(kStages - 1, kStages - 1);
      Half h0, h1;
      read_half(jt, 0, 0, h0);
      for (int s = 0; s < KT; ++s) {
        const int buf = s % kStages;
        // Phase A: the kk = 0 MFMAs of stage s, with the kk = 1 fragment
        // reads of the same stage slotted between them.
        read_half(jt, buf, 1, h1);
        mfma_half(jt, h0);
#pragma unroll
        for (int q = 0; q < 4 + JT; ++q) {
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
        }
        __builtin_amdgcn_sched_group_barrier(0x008, NM - 4 - JT, 0);
        __builtin_amdgcn_sched_barrier(0);
        if (s + 1 < KT) {
          wait_vm(min(kStages - 2, KT - 2 - s));
          asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // this wave's reads of stage s are done
          barrier_nofence();
          if (s + kStages < KT) issue_stage(s + kStages, buf);
          read_half(jt, (s + 1) % kStages, 0, h0);
        }
        // Phase B: the kk = 1 MFMAs, with the kk = 0 fragment reads of stage
        // s + 1 slotted between them (the copies of stage s + kStages go first).
        mfma_half(jt, h1);
#pragma unroll
        for (int q = 0; q < 4 + JT; ++q) {
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 1);  // one LDS read
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 1);  // one MFMA
        }
        __builtin_amdgcn_sched_group_barrier(0x008, NM - 4 - JT, 1);
        __builtin_amdgcn_sched_barrier(0);
      }
    };
    if (hm < 0)
      k_loop(std::integral_constant<int, 4>{});
    else
      k_loop(std::integral_constant<int, 2>{});

    // All waves are done with every stage: start the next tile's copies so
    // they overlap this tile's epilogue.
    const int L_next = L + G;
    __syncthreads();
    if (L_next < n_units) {
      int nm, nn, nh;
      unit_coords(L_next, nm, nn, nh);
      set_tile(nm, nn, nh);
#pragma unroll
      for (int st = 0; st < kStages - 1; ++st)
        if (st < KT) issue_stage(st, st);
    }

    // ---------------------------------------------------------------- epilogue
    const int nj = hm < 0 ? 4 : 2;
    const int m0 = tile_m * BM + (hm < 0 ? wm * 128 : hm * 128 + wm * 64) + fr;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int m = m0 + j * 32;
      if (j >= nj || m >= a.M) continue;
      if constexpr (EPI == EPI_RESID) {
        // out (fp32) = resid (bf16 or fp32) + acc: the residual stream stays in fp32.
        const int n_base = tile_n * BN + wn * 128 + 4 * fh;
        float* orow = a.out_f32 + int64_t(m) * a.ldo;
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const int n = n_base + i * 32 + 8 * g;
            f32x4 v = {acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]};
            if (a.resid_f32) {
              const f32x4 r = *reinterpret_cast<const f32x4*>(a.resid_f32 + int64_t(m) * a.ldo + n);
              v += r;
            } else {
              float r[4];
              load_bf16x4(a.resid + int64_t(m) * a.ldo + n, r);
              v[0] += r[0];
              v[1] += r[1];
              v[2] += r[2];
              v[3] += r[3];
            }
            *reinterpret_cast<f32x4*>(orow + n) = v;
          }
      } else if constexpr (EPI == EPI_SWIGLU) {
        const int c_base = tile_n * 128 + wn * 64 + 4 * fh;
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            float v[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = silu(acc[i][j][4 * g + e]) * acc[i + 2][j][4 * g + e];
            store_h4(a.out + int64_t(m) * a.ldo + c_base + i * 32 + 8 * g, v[0], v[1], v[2], v[3]);
          }
      } else {  // EPI_QKV
        const int p = a.pos[m];
        const float2* rt = a.rope + int64_t(p) * (DH / 2);
#pragma unroll
        for (int pr = 0; pr < 2; ++pr) {  // (lo subtile, hi subtile) pairs of the wave
          // DH 128: one head per wave, pairs (0, 2), (1, 3); d_lo = 32 pr + ...
          // DH  64: two heads per wave, pairs (0, 1), (2, 3); d_lo = ...
          const int lo_i = (DH == 128) ? pr : 2 * pr;
          const int hi_i = (DH == 128) ? pr + 2 : 2 * pr + 1;
          const int head = (tile_n * BN + wn * 128) / DH + ((DH == 128) ? 0 : pr);
          const int dsub = (DH == 128) ? 32 * pr : 0;
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const int d = dsub + 8 * g + 4 * fh;  // < DH / 2
            float lo[4], hi[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              lo[e] = acc[lo_i][j][4 * g + e];
              hi[e] = acc[hi_i][j][4 * g + e];
            }
            if (head < a.hq + a.hkv) {
              float rl[4], rh[4];
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                const float2 cs = rt[d + e];
                rl[e] = lo[e] * cs.x - hi[e] * cs.y;
                rh[e] = hi[e] * cs.x + lo[e] * cs.y;
              }
              uint16_t* dst = (head < a.hq)
                                  ? a.q + (int64_t(m) * a.hq + head) * DH
                                  : a.kstore + a.k_off[m] + int64_t(head - a.hq) * DH;
              store_h4(dst + d, rl[0], rl[1], rl[2], rl[3]);
              store_h4(dst + d + DH / 2, rh[0], rh[1], rh[2], rh[3]);
            } else {
              const int gh = head - a.hq - a.hkv;
              uint16_t* dst = a.vstore + a.v_off[m];
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                dst[int64_t(gh * DH + d + e) * a.v_stride] = f2h(lo[e]);
                dst[int64_t(gh * DH + d + DH / 2 + e) * a.v_stride] = f2h(hi[e]);
              }
            }
          }
        }
      }
    }
    if (L_next >= n_units) break;
    L = L_next;
    unit_coords(L, tile_m, tile_n, hm);
  }
}

template <int EPI, int DH>
hipError_t launch_one(const GemmArgs& a, int max_blocks, hipStream_t s) {
  const int n_tiles = ((a.M + BM - 1) / BM) * a.n_tiles_n;
  int grid = n_tiles < max_blocks ? n_tiles : max_blocks;
  if (grid < 1) return hipSuccess;
  if (a.w_f16)
    hipLaunchKernelGGL((gemm_kernel<EPI, DH, true>), dim3(grid), dim3(kThreads), 0, s, a);
  else
    hipLaunchKernelGGL((gemm_kernel<EPI, DH, false>), dim3(grid), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm(int epi, const GemmArgs& a, int max_blocks, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  switch (epi) {
    case EPI_RESID: return launch_one<EPI_RESID, 128>(a, max_blocks, s);
    case EPI_SWIGLU: return launch_one<EPI_SWIGLU, 128>(a, max_blocks, s);
    case EPI_QKV:
      return a.dh == 64 ? launch_one<EPI_QKV, 64>(a, max_blocks, s)
                        : launch_one<EPI_QKV, 128>(a, max_blocks, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace hs
