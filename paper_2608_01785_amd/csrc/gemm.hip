// Persistent fp16 MFMA GEMM for gfx950 with fused epilogues.
//
// Computes C[M, N] = A[M, K] * W[N, K]^T (fp16 activations times bf16 [out, in]
// weights, fp32 accumulation).  Weight tiles are converted bf16 -> fp16 on
// their way into LDS (exact for the weight range), so both MFMA operands are
// fp16: the same MFMA rate as bf16 on gfx950 with 8x finer rounding of the
// activations.  The MFMA is issued as C^T = W * A^T: the weight tile is the MFMA
// A operand and the activation tile the B operand, so every lane of the 32x32
// accumulator owns one activation row and four consecutive output columns per
// register group.  That makes 8-byte output stores possible and keeps the
// pairs the epilogues need (RoPE's (j, j + dh/2), SwiGLU's gate/up) in the
// same lane and register.
//
// Block tile 256 (weight rows) x 256 (activation rows) x 64 (K), 4 waves in a
// 2 x 2 grid, each wave 128 x 128 = 4 x 4 MFMA tiles of 32x32x16.  Operands go
// global -> registers -> LDS (two stages, XOR-swizzled 16-byte chunks) and
// the next K slab is fetched while the current one feeds the MFMAs.  The grid
// is persistent (at most one block per CU of the budget); blocks walk the
// tile space in grouped order, remapped so each XCD takes a contiguous range.
#include "hs_device.h"
#include "hs_kernels.h"

namespace hs {
namespace {

constexpr int BM = 256;   // activation rows per tile
constexpr int BN = 256;   // weight rows per tile
constexpr int BK = 64;
constexpr int kThreads = 256;
constexpr int kRowBytes = BK * 2;            // 128 bytes = 8 chunks of 16
constexpr int kTileBytes = 256 * kRowBytes;  // 32 KB
constexpr int kStageBytes = 2 * kTileBytes;  // weight tile + activation tile
constexpr int kGroupM = 8;

template <int EPI>
__device__ __forceinline__ int64_t weight_row(int tile_n, int j, int ld_row, int ffn) {
  // Row of W loaded into tile row ld_row + 32 j.
  if constexpr (EPI == EPI_SWIGLU) {
    // Tile rows: [wave-n 0: gate 64 | up 64][wave-n 1: gate 64 | up 64] for
    // output columns tile_n * 128 .. +128.
    const int half = j >> 2;            // which wave-n half (rows 128 * half ..)
    const int up = (j & 3) >> 1;        // rows 64..127 of the half are 'up'
    const int jj = ld_row + 32 * (j & 1);
    return int64_t(up) * ffn + tile_n * 128 + half * 64 + jj;
  } else {
    return int64_t(tile_n) * BN + ld_row + 32 * j;
  }
}

__device__ __forceinline__ float silu(float z) { return z / (1.0f + __expf(-z)); }

template <int EPI, int DH>
__global__ __launch_bounds__(kThreads, 1) void gemm_kernel(GemmArgs a) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[2 * kStageBytes];

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
  const int ld_row = tid >> 3;   // 0..31
  const int ld_chunk = tid & 7;
  const int ld_phys = ld_chunk ^ (ld_row & 7);  // rows ld_row + 32 j share (row & 7)

  const int per_group = kGroupM * a.n_tiles_n;
  for (int L = xcd_remap(blockIdx.x, gridDim.x); L < n_tiles; L += gridDim.x) {
    const int group = L / per_group;
    const int first_m = group * kGroupM;
    const int gsize = min(n_m_tiles - first_m, kGroupM);
    const int tile_m = first_m + (L % per_group) % gsize;
    const int tile_n = (L % per_group) / gsize;

    // Weight rows of one thread differ by wave-uniform offsets (scalar registers);
    // activation rows are clamped to the last valid row in a ragged tail tile.
    const uint16_t* wsrc = a.W + weight_row<EPI>(tile_n, 0, ld_row, a.ffn) * a.K + ld_chunk * 8;
    const int arow0 = tile_m * BM + ld_row;
    const bool a_full = tile_m * BM + BM <= a.M;
    const uint16_t* asrc = a.A + int64_t(arow0) * a.K + ld_chunk * 8;

    u32x4 rw[8], ra[8];
    auto gload = [&](int kt) {
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int64_t wofs = (weight_row<EPI>(tile_n, j, 0, a.ffn) - weight_row<EPI>(tile_n, 0, 0, a.ffn)) * a.K;
        rw[j] = *reinterpret_cast<const u32x4*>(wsrc + wofs + kt * BK);
        const int64_t arow = a_full ? int64_t(32 * j) : int64_t(min(arow0 + 32 * j, a.M - 1) - arow0);
        ra[j] = *reinterpret_cast<const u32x4*>(asrc + arow * a.K + kt * BK);
      }
    };
    auto lstore = [&](int stage) {
      uint8_t* base = smem + stage * kStageBytes;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int off = (ld_row + 32 * j) * kRowBytes + ld_phys * 16;
        *reinterpret_cast<u32x4*>(base + off) = bf8_to_h8(rw[j]);
        *reinterpret_cast<u32x4*>(base + kTileBytes + off) = ra[j];
      }
    };

    f32x16 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    gload(0);
    lstore(0);
    __syncthreads();

    for (int kt = 0; kt < KT; ++kt) {
      const int cur = kt & 1;
      if (kt + 1 < KT) gload(kt + 1);
      const uint8_t* base = smem + cur * kStageBytes;
#pragma unroll
      for (int kk = 0; kk < BK / 16; ++kk) {
        const int phys = (kk * 2 + fh) ^ (fr & 7);
        u32x4 wf[4], af[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
          wf[i] = *reinterpret_cast<const u32x4*>(base + (wn * 128 + i * 32 + fr) * kRowBytes + phys * 16);
#pragma unroll
        for (int j = 0; j < 4; ++j)
          af[j] = *reinterpret_cast<const u32x4*>(base + kTileBytes + (wm * 128 + j * 32 + fr) * kRowBytes + phys * 16);
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[i][j] = mfma32(wf[i], af[j], acc[i][j]);
      }
      if (kt + 1 < KT) lstore(cur ^ 1);
      __syncthreads();
    }

    // ---------------------------------------------------------------- epilogue
    const int m0 = tile_m * BM + wm * 128 + fr;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int m = m0 + j * 32;
      if (m >= a.M) continue;
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
  }
}

template <int EPI, int DH>
hipError_t launch_one(const GemmArgs& a, int max_blocks, hipStream_t s) {
  const int n_tiles = ((a.M + BM - 1) / BM) * a.n_tiles_n;
  int grid = n_tiles < max_blocks ? n_tiles : max_blocks;
  if (grid < 1) return hipSuccess;
  hipLaunchKernelGGL((gemm_kernel<EPI, DH>), dim3(grid), dim3(kThreads), 0, s, a);
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
