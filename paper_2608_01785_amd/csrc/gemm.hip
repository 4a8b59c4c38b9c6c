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
// Block tile 256 (weight rows) x 256 (activation rows), 8 waves (two per
// SIMD) in a 2 x 4 grid, each wave 128 weight rows x 64 activation rows =
// 4 x 2 MFMA tiles of 32x32x16.  K advances in stages of 32.
//
// Operand staging.  Copies straight from the buffer unit into LDS occupy the
// LDS for far longer per byte than ds_write_b128 and serialise with the
// fragment reads, and a wave can keep only a few vector-memory instructions
// moving at a time.  So each stage is fetched with plain 16-byte loads into a
// ring of registers (waves 0-3 the weight tile, waves 4-7 the activation
// tile, 4 x 1 KB per wave) and written to LDS by the same wave:
//   stage t is loaded during stage t - 4, written to LDS buffer t % 2 in the
//   first half of stage t - 1 and multiplied during stage t.
// One barrier per stage, between its two 16-wide halves, after each wave's
// writes of stage t + 1 and fragment reads of stage t have completed: that
// makes the writes visible to the second half's reads of stage t + 1 and
// retires every read of the buffer the next stage overwrites.  K must be a
// multiple of 128, so every tile starts on buffer 0 and register slot 0, and
// the loads of a tile's last four stages already fetch the next tile's first
// four: the pipeline runs across tiles and the epilogue overlaps them.
//
// The grid is persistent (one block per CU of the budget); blocks walk the
// tile space in grouped order, remapped so each XCD takes a contiguous range,
// and in alternating block order from round to round.
#include <type_traits>

#include "hs_device.h"
#include "hs_kernels.h"

namespace hs {
namespace {

constexpr int BM = 256;   // activation rows per tile
constexpr int BN = 256;   // weight rows per tile
constexpr int BK = 32;    // K per stage
constexpr int kThreads = 512;
constexpr int kRowBytes = BK * 2;            // 64 bytes = 4 chunks of 16
constexpr int kTileBytes = 256 * kRowBytes;  // 16 KB
constexpr int kStageBytes = 2 * kTileBytes;  // weight tile + activation tile
constexpr int kLoads = 4;                    // 1 KB loads per wave per stage
constexpr int kUnroll = 4;                   // stages per loop body
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

// 16-byte chunk c of tile row r sits at physical chunk c ^ swz(r).  A
// 16-lane pass of fragment reads covers rows r0 .. r0 + 15 at one logical
// chunk; (r & 3, c ^ swz(r)) is then distinct for all 16 rows, so the pass
// touches each of the 64 banks once (and any 8 consecutive rows each of 32).
__device__ __forceinline__ int swz(int r) { return ((r >> 1) ^ (r >> 2)) & 3; }

// silu(z) = z / (1 + e^-z), with the hardware reciprocal (1 ulp) in place of
// an IEEE division: the result is rounded to fp16 next.
__device__ __forceinline__ float silu(float z) { return z * __builtin_amdgcn_rcpf(1.0f + __expf(-z)); }

// Buffer resource over [base, base + bytes): loads past the end return zero.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, 0x00020000);
}

template <int EPI, int DH, bool W_F16>
__global__ __launch_bounds__(kThreads, 1) void gemm_kernel(GemmArgs a) {
  __shared__ __attribute__((aligned(1024))) uint8_t smem[2 * kStageBytes];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  LaunchClock clk;
  clk.begin(a.clock);
  const int wn = wave & 1;   // weight-row half of the tile (128 rows)
  const int wm = wave >> 1;  // activation-row quarter (64 rows; 32 in a half unit)
  const int fr = lane & 31;
  const int fh = lane >> 5;

  const int n_m_tiles = (a.M + BM - 1) / BM;
  const int n_tiles = n_m_tiles * a.n_tiles_n;
  const int KT = a.K / BK;
  const uint32_t row_bytes = uint32_t(a.K) * 2;
  const uint32_t w_rows = (EPI == EPI_SWIGLU) ? uint32_t(2 * a.ffn) : uint32_t(a.n_tiles_n * BN);

  // Loads: waves 0-3 fetch the weight tile, waves 4-7 the activation tile.
  // Load l of a wave covers tile rows 64 (wave % 4) + 16 l .. + 15; lane i
  // fetches chunk i % 4 of row 16 l + i / 4 and writes it to LDS at its
  // swizzled position.
  const bool w_wave = wave < 4;
  const __amdgpu_buffer_rsrc_t res =
      w_wave ? make_rsrc(a.W, w_rows * row_bytes) : make_rsrc(a.A, uint32_t(a.M) * row_bytes);
  // Bytes between consecutive stages of one row.  fp16 weights are
  // panel-major ([K / 32][N][32]): a stage of a weight row is 64 contiguous
  // bytes and the next stage w_rows * 64 bytes further on.
  const uint32_t kstride = (w_wave && W_F16) ? w_rows * kRowBytes : uint32_t(kRowBytes);
  const int ld_sub = lane >> 2;
  const int ld_chunk = lane & 3;
  const int lrow0 = (wave & 3) * 64 + ld_sub;
  uint32_t off[kLoads];
  // A half unit (hm = 0 or 1) covers activation rows hm * 128 .. + 127 of
  // its tile: LDS activation rows 0..127 hold them.  Waves 6 and 7 still
  // issue their four loads per stage (the pipeline's counts stay uniform),
  // but at an offset past the buffer's end, like rows >= M: those loads
  // return zeros into the unused rows 128..255 and move no data.
  auto set_loads = [&](int tile_m, int tile_n, int hm) {
#pragma unroll
    for (int l = 0; l < kLoads; ++l) {
      const int r = lrow0 + 16 * l;
      if (w_wave) {
        off[l] = weight_row<EPI>(tile_n, r, a.ffn) * (W_F16 ? uint32_t(kRowBytes) : row_bytes) + ld_chunk * 16;
      } else if (hm >= 0 && r >= 128) {
        off[l] = uint32_t(a.M) * row_bytes + ld_chunk * 16;
      } else {
        const int ar = hm < 0 ? r : hm * 128 + r;
        off[l] = uint32_t(tile_m * BM + ar) * row_bytes + ld_chunk * 16;  // rows >= M read zero
      }
    }
  };
  const uint32_t wr_off = (w_wave ? 0u : uint32_t(kTileBytes)) + uint32_t(lrow0 * kRowBytes) +
                          uint32_t((ld_chunk ^ swz(ld_sub)) * 16);

  u32x4 g[kUnroll][kLoads];  // register ring: stage t in slot t % 4
  auto gload = [&](int kt, u32x4* dst) {
    const uint32_t so = uint32_t(kt) * kstride;
#pragma unroll
    for (int l = 0; l < kLoads; ++l)
      dst[l] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(res, off[l], so, 0));
  };
  auto lwrite = [&](int buf, const u32x4* v) {
    uint8_t* base = smem + buf * kStageBytes + wr_off;
#pragma unroll
    for (int l = 0; l < kLoads; ++l) *reinterpret_cast<u32x4*>(base + l * 16 * kRowBytes) = v[l];
  };

  // Fragments of one 16-wide half stage: [i] weight subtile, [j] activation
  // subtile.  JT = activation subtiles per wave: 2 (full tile) or 1 (half unit).
  struct Frag {
    u32x4 w[4], a[2];
  };
  auto read_frag = [&](auto jt, int buf, int kk, Frag& h) {
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

  // Work units.  When the last M-tile holds at most 128 rows, its tiles are
  // half units (rows 0..127 of the tile, hm = 0) placed after all others.
  // The other tiles are full units, except that when their last round would
  // leave more than half the blocks idle (counting the short tiles' halves)
  // its tiles are split into two 128-row halves.  Each output element is
  // accumulated in the same order either way, so the result does not depend
  // on the grid.
  const bool short_last = a.M - (n_m_tiles - 1) * BM <= 128;
  const int n_m_full = short_last ? n_m_tiles - 1 : n_m_tiles;
  const int n_full = n_m_full * a.n_tiles_n;
  const int n_short = short_last ? a.n_tiles_n : 0;
  const int per_group = kGroupM * a.n_tiles_n;
  auto tile_coords = [&](int L, int& tile_m, int& tile_n) {
    const int group = L / per_group;
    const int first_m = group * kGroupM;
    const int gsize = min(n_m_full - first_m, kGroupM);
    tile_m = first_m + (L % per_group) % gsize;
    tile_n = (L % per_group) / gsize;
  };
  const int G = gridDim.x;
  const int full_units = (n_full / G) * G;
  const int tail = n_full - full_units;
  const bool split_tail = tail > 0 && 2 * tail + n_short <= G;
  const int n_split = split_tail ? full_units + 2 * tail : n_full;
  const int n_units = n_split + n_short;
  auto unit_coords = [&](int u, int& tile_m, int& tile_n, int& hm) {
    if (u >= n_split) {
      tile_m = n_m_tiles - 1;
      tile_n = u - n_split;
      hm = 0;
      return;
    }
    int t = u;
    hm = -1;
    if (split_tail && u >= full_units) {
      t = full_units + (u - full_units) / 2;
      hm = (u - full_units) % 2;
    }
    tile_coords(t, tile_m, tile_n);
  };

  // Round r gives block b unit r G + b, or r G + G - 1 - b in odd rounds: the
  // blocks left without a full tile in a round take the first halves of the
  // next.  Every round still covers a contiguous range of units, split over
  // the XCDs in contiguous pieces.
  const int b = xcd_remap(blockIdx.x, G);
  auto unit_of = [&](int r) { return r * G + ((r & 1) ? G - 1 - b : b); };
  int round = 0;
  int L = unit_of(0);
  if (L >= n_units) return;
  int tile_m, tile_n, hm;
  unit_coords(L, tile_m, tile_n, hm);
  set_loads(tile_m, tile_n, hm);
#pragma unroll
  for (int q = 0; q < kUnroll; ++q) gload(q, g[q]);
  lwrite(0, g[0]);
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();

  f32x16 acc[4][2];
  while (true) {
    // Output rows of this lane: m0 + 32 j for j < nj.
    const int nj = hm < 0 ? 2 : 1;
    const int m0 = tile_m * BM + (hm < 0 ? wm * 64 : hm * 128 + wm * 32) + fr;
    const int L_next = unit_of(round + 1);

    auto mfma_half = [&](auto jt, const Frag& h) {
      constexpr int JT = decltype(jt)::value;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const u32x4 wh = W_F16 ? h.w[i] : bf8_to_h8(h.w[i]);
#pragma unroll
        for (int j = 0; j < JT; ++j) acc[i][j] = mfma32(wh, h.a[j], acc[i][j]);
      }
    };

    // Accumulator start values for a unit with JT activation subtiles per
    // wave (the rows a half unit does not own stay constant zeros).
    auto init_acc = [&](auto jt) {
      constexpr int JT = decltype(jt)::value;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;
      if constexpr (EPI == EPI_RESID) {
        // The accumulators start from the residual, so the epilogue is plain
        // stores: these loads overlap the previous unit's stores and this
        // unit's first stages instead of stalling a separate epilogue pass.
        // Rows past M (never stored) read the last valid row instead.
        const int n_base = tile_n * BN + wn * 128 + 4 * fh;
        int64_t roff[JT];
#pragma unroll
        for (int j = 0; j < JT; ++j) roff[j] = int64_t(min(m0 + j * 32, a.M - 1)) * a.ldo + n_base;
        if (a.resid_f32) {
#pragma unroll
          for (int j = 0; j < JT; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
              for (int g4 = 0; g4 < 4; ++g4) {
                const f32x4 v = *reinterpret_cast<const f32x4*>(a.resid_f32 + roff[j] + i * 32 + 8 * g4);
#pragma unroll
                for (int e = 0; e < 4; ++e) acc[i][j][4 * g4 + e] = v[e];
              }
        } else {
#pragma unroll
          for (int j = 0; j < JT; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
              for (int g4 = 0; g4 < 4; ++g4) {
                float r[4];
                load_bf16x4(a.resid + roff[j] + i * 32 + 8 * g4, r);
#pragma unroll
                for (int e = 0; e < 4; ++e) acc[i][j][4 * g4 + e] = r[e];
              }
        }
      }
    };
    // Stage s of the unit: buffer s % 2, register slot s % 4 (K % 128 == 0).
    auto k_loop = [&](auto jt) {
      constexpr int JT = decltype(jt)::value;
      constexpr int NM = 4 * JT;      // MFMAs per half stage
      constexpr int NR = 4 + JT;      // fragment reads per half stage
      Frag h0, h1;
      init_acc(jt);
      read_frag(jt, 0, 0, h0);
      for (int kt = 0; kt < KT; kt += kUnroll) {
        const bool last = kt + kUnroll == KT;
        if (last && L_next < n_units) {
          // The loads of this body fetch the next unit's first four stages.
          int nm, nn, nh;
          unit_coords(L_next, nm, nn, nh);
          set_loads(nm, nn, nh);
        }
        // After the last unit the loads repeat its first stages (in bounds,
        // never used).
        const int kl = last ? 0 : kt + kUnroll;
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
          // First half: the kk = 0 MFMAs of stage s, with the LDS writes of
          // stage s + 1, the loads of stage s + 4 and the kk = 1 fragment
          // reads of stage s slotted between them.
          read_frag(jt, u & 1, 1, h1);
          lwrite((u + 1) & 1, g[(u + 1) & 3]);
          gload(kl + u, g[u]);
          mfma_half(jt, h0);
          // LDS traffic first (the barrier below waits for it), then the
          // loads, one per MFMA.
#pragma unroll
          for (int q = 0; q < kLoads; ++q) {
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
            __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);  // one LDS write
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
          }
#pragma unroll
          for (int q = kLoads; q < NR; ++q) {
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
            __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // one load
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
          }
#pragma unroll
          for (int q = NR - kLoads; q < kLoads; ++q) {
            __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // one load
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
          }
          __builtin_amdgcn_sched_barrier(0);
          // Writes of stage s + 1 and reads of stage s are done on this
          // wave; after the barrier on every wave.
          asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
          __builtin_amdgcn_s_barrier();
          // Second half: the kk = 1 MFMAs, with the kk = 0 fragment reads of
          // stage s + 1 (the next unit re-reads its own first fragments).
          if (u + 1 < kUnroll || !last) read_frag(jt, (u + 1) & 1, 0, h0);
          mfma_half(jt, h1);
#pragma unroll
          for (int q = 0; q < NR; ++q) {
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 1);  // one LDS read
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 1);  // one MFMA
          }
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      (void)NM;
    };
    if (hm < 0)
      k_loop(std::integral_constant<int, 2>{});
    else
      k_loop(std::integral_constant<int, 1>{});

    // ---------------------------------------------------------------- epilogue
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int m = m0 + j * 32;
      if (j >= nj || m >= a.M) continue;
      if constexpr (EPI == EPI_RESID) {
        // out (fp32) = resid + products, the accumulators having started from
        // the residual: the residual stream stays in fp32.
        const int n_base = tile_n * BN + wn * 128 + 4 * fh;
        float* orow = a.out_f32 + int64_t(m) * a.ldo;
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const int n = n_base + i * 32 + 8 * g;
            const f32x4 v = {acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]};
            *reinterpret_cast<f32x4*>(orow + n) = v;
          }
      } else if constexpr (EPI == EPI_GATED) {
        // out (fp32) = resid + gate_seq(m) * (products + bias): the adaLN-Zero
        // residual branch.  Stores count against the same completion counter
        // as loads, so each group's operands are loaded before the previous
        // group's store: waiting for them never waits for a store.
        const int n_base = tile_n * BN + wn * 128 + 4 * fh;
        float* orow = a.out_f32 + int64_t(m) * a.ldo + n_base;
        const float* grow = a.gate + int64_t(a.row_seq[m]) * a.gate_stride + n_base;
        const float* rrow = a.resid_f32 ? a.resid_f32 + int64_t(m) * a.ldo + n_base : nullptr;
        const uint16_t* rrow16 = a.resid + int64_t(m) * a.ldo + n_base;
        const uint16_t* brow = a.bias + n_base;
        struct Ops {
          u32x2 b;
          f32x4 r, gt;
        };
        auto load_ops = [&](int q) {
          const int c = (q >> 2) * 32 + 8 * (q & 3);
          Ops o;
          o.b = *reinterpret_cast<const u32x2*>(brow + c);
          if (rrow) {
            o.r = *reinterpret_cast<const f32x4*>(rrow + c);
          } else {
            const u32x2 r2 = *reinterpret_cast<const u32x2*>(rrow16 + c);
            o.r = f32x4{__uint_as_float(r2.x << 16), __uint_as_float(r2.x & 0xffff0000u), __uint_as_float(r2.y << 16),
                        __uint_as_float(r2.y & 0xffff0000u)};
          }
          o.gt = *reinterpret_cast<const f32x4*>(grow + c);
          return o;
        };
        Ops nx = load_ops(0);
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          const int i = q >> 2, g = q & 3;
          const Ops cur = nx;
          if (q + 1 < 16) nx = load_ops(q + 1);
          const float b4[4] = {__uint_as_float(cur.b.x << 16), __uint_as_float(cur.b.x & 0xffff0000u),
                               __uint_as_float(cur.b.y << 16), __uint_as_float(cur.b.y & 0xffff0000u)};
          f32x4 v;
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = cur.r[e] + cur.gt[e] * (acc[i][j][4 * g + e] + b4[e]);
          *reinterpret_cast<f32x4*>(orow + i * 32 + 8 * g) = v;
        }
      } else if constexpr (EPI == EPI_GELU) {
        // out (fp16) = gelu_tanh(products + bias); 0.5 z (1 + tanh(u)) = z / (1 + exp(-2u))
        // with u = sqrt(2 / pi) (z + 0.044715 z^3), and exp(-2u) = 2^(z (k1 + k2 z^2)),
        // k1 = -2 sqrt(2 / pi) log2(e), k2 = 0.044715 k1.  Groups 2p and 2p + 1
        // are stored as one 32-byte run of the row, and each pair's bias is
        // loaded before the previous pair's store: stores count against the
        // same completion counter as loads, so waiting for it never waits for
        // a store.
        constexpr float k1 = -2.302208198144325f, k2 = -0.1029432395800235f;
        const int n_base = tile_n * BN + wn * 128;
        uint16_t* orow = a.out + int64_t(m) * a.ldo + n_base;
        const uint16_t* brow = a.bias + n_base + 4 * fh;
        auto load_bias = [&](int q) {  // bias of group q of this lane
          return *reinterpret_cast<const u32x2*>(brow + (q >> 2) * 32 + 8 * (q & 3));
        };
        u32x2 bnext[2] = {load_bias(0), load_bias(1)};
#pragma unroll
        for (int qp = 0; qp < 8; ++qp) {
          const int i = qp >> 1, p = qp & 1;
          const u32x2 b[2] = {bnext[0], bnext[1]};
          if (qp + 1 < 8) {
            bnext[0] = load_bias(2 * qp + 2);
            bnext[1] = load_bias(2 * qp + 3);
          }
          float v[2][4];
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const float b4[4] = {__uint_as_float(b[h].x << 16), __uint_as_float(b[h].x & 0xffff0000u),
                                 __uint_as_float(b[h].y << 16), __uint_as_float(b[h].y & 0xffff0000u)};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const float z = acc[i][j][8 * p + 4 * h + e] + b4[e];
              v[h][e] = z * __builtin_amdgcn_rcpf(1.0f + exp2_raw(z * fmaf(z * z, k2, k1)));
            }
          }
          store_h8_pair(orow + i * 32 + 16 * p, fh, v[0], v[1]);
        }
      } else if constexpr (EPI == EPI_SWIGLU) {
        // Groups 2p and 2p + 1 are stored as one 32-byte run of the row.
        uint16_t* orow = a.out + int64_t(m) * a.ldo + tile_n * 128 + wn * 64;
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int p = 0; p < 2; ++p) {
            float lo[4], hi[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              lo[e] = silu(acc[i][j][8 * p + e]) * acc[i + 2][j][8 * p + e];
              hi[e] = silu(acc[i][j][8 * p + 4 + e]) * acc[i + 2][j][8 * p + 4 + e];
            }
            store_h8_pair(orow + i * 32 + 16 * p, fh, lo, hi);
          }
      } else {  // EPI_QKV
        // The row's positions (one per RoPE section) and cache offsets, loaded
        // once per row rather than once per four pairs.
        const bool sectioned = a.pos_stride != 0;
        const int p0 = a.pos[m];
        const int p1 = sectioned ? a.pos[a.pos_stride + m] : p0;
        const int p2 = sectioned ? a.pos[2 * a.pos_stride + m] : p0;
        const int64_t k_row = a.k_off[m], v_row = a.v_off[m];
#pragma unroll
        for (int pr = 0; pr < 2; ++pr) {  // (lo subtile, hi subtile) pairs of the wave
          // DH 128: one head per wave, pairs (0, 2), (1, 3); d_lo = 32 pr + ...
          // DH  64: two heads per wave, pairs (0, 1), (2, 3); d_lo = ...
          const int lo_i = (DH == 128) ? pr : 2 * pr;
          const int hi_i = (DH == 128) ? pr + 2 : 2 * pr + 1;
          const int head = (tile_n * BN + wn * 128) / DH + ((DH == 128) ? 0 : pr);
          const int dsub = (DH == 128) ? 32 * pr : 0;
          // Q and K: groups 2p and 2p + 1 are stored as one 32-byte run of
          // each half of the head.
#pragma unroll
          for (int p = 0; p < 2; ++p) {
            float rl[2][4], rh[2][4];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
              const int g = 2 * p + h;
              const int d = dsub + 8 * g + 4 * fh;  // < DH / 2
              // Pairs d .. d + 3 share one RoPE section (sections are multiples of 4 pairs).
              const int pc = d >= a.sec2 ? p2 : (d >= a.sec1 ? p1 : p0);
              const float2* rt = a.rope ? a.rope + int64_t(pc) * (DH / 2) : nullptr;
              float lo[4], hi[4];
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                lo[e] = acc[lo_i][j][4 * g + e];
                hi[e] = acc[hi_i][j][4 * g + e];
              }
              if (a.bias) {
                float bl[4], bh[4];
                load_bf16x4(a.bias + head * DH + d, bl);
                load_bf16x4(a.bias + head * DH + d + DH / 2, bh);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                  lo[e] += bl[e];
                  hi[e] += bh[e];
                }
              }
              if (head < a.hq + a.hkv) {
                if (a.rope) {
#pragma unroll
                  for (int e = 0; e < 4; ++e) {
                    const float2 cs = rt[d + e];
                    rl[h][e] = lo[e] * cs.x - hi[e] * cs.y;
                    rh[h][e] = hi[e] * cs.x + lo[e] * cs.y;
                  }
                } else {
#pragma unroll
                  for (int e = 0; e < 4; ++e) {
                    rl[h][e] = lo[e];
                    rh[h][e] = hi[e];
                  }
                }
              } else {
                const int gh = head - a.hq - a.hkv;
                uint16_t* dst = a.vstore + v_row + int64_t(gh) * a.kv_head_stride;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                  dst[(d + e) * kv_tile_keys] = f2h(lo[e]);
                  dst[(d + DH / 2 + e) * kv_tile_keys] = f2h(hi[e]);
                }
              }
            }
            if (head < a.hq + a.hkv) {
              uint16_t* dst = (head < a.hq)
                                  ? a.q + (int64_t(m) * a.hq + head) * DH
                                  : a.kstore + k_row + int64_t(head - a.hq) * a.kv_head_stride;
              store_h8_pair(dst + dsub + 16 * p, fh, rl[0], rl[1]);
              store_h8_pair(dst + dsub + 16 * p + DH / 2, fh, rh[0], rh[1]);
            }
          }
        }
      }
    }
    if (L_next >= n_units) break;
    L = L_next;
    ++round;
    unit_coords(L, tile_m, tile_n, hm);
  }
  clk.end(a.clock);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
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
  if (a.K < BK * kUnroll || a.K % (BK * kUnroll) != 0) return hipErrorInvalidValue;
  if (a.sumsq_out || a.scaled_out || a.row_sumsq) return hipErrorInvalidValue;
  switch (epi) {
    case EPI_RESID: return launch_one<EPI_RESID, 128>(a, max_blocks, s);
    case EPI_SWIGLU: return launch_one<EPI_SWIGLU, 128>(a, max_blocks, s);
    case EPI_GATED: return launch_one<EPI_GATED, 128>(a, max_blocks, s);
    case EPI_GELU: return launch_one<EPI_GELU, 128>(a, max_blocks, s);
    case EPI_QKV:
      return a.dh == 64 ? launch_one<EPI_QKV, 64>(a, max_blocks, s)
                        : launch_one<EPI_QKV, 128>(a, max_blocks, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace hs
