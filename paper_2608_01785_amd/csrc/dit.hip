// Diffusion-transformer pieces for gfx950: the adaLN modulation of each
// sequence and the modulated LayerNorm that feeds a block's QKV and MLP
// GEMMs.  The projections themselves run on the persistent GEMM (gemm.hip)
// with its bias + gated-residual and bias + GELU epilogues, and attention on
// the prefill kernel in its bidirectional mode.
#include "hs_device.h"
#include "hs_kernels.h"

namespace hs {
namespace {

constexpr int kMaxChunksPerLane = 16;  // d <= 64 lanes * 16 chunks * 8 = 8192

__global__ __launch_bounds__(256) void silu_rows_kernel(const float* __restrict__ c, float* __restrict__ s, int n) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
    const float z = c[i];
    s[i] = z / (1.0f + __expf(-z));
  }
}

// The modulation of up to kDitModLayers layers in one launch (it depends on
// the conditioning only, not on the layer's input).  Each wave takes RW
// consecutive rows j of one layer's W (bf16 [6d, d]) with every load in
// flight at once, then takes their dot products with each sequence's
// silu(c) (fp32, L2-resident): mod[l][b][j] = bias_l[j] + sum_k s[b][k] W_l[j][k].
// CPL = 16-byte chunks per lane (d <= 512 CPL).
template <int CPL, int RW>
__global__ __launch_bounds__(256) void dit_mod_kernel(DitModArgs p, const float* __restrict__ s,
                                                      float* __restrict__ mod, int n_seqs, int d) {
  const int lane = threadIdx.x & 63;
  const int rows = 6 * d;
  const int64_t row0 = (int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6)) * RW;
  if (row0 >= int64_t(p.n_layers) * rows) return;
  const int l = int(row0 / rows), j0 = int(row0 % rows);  // RW divides rows
  const int chunks = d >> 3;
  const uint16_t* wl = p.w[l];
  u32x4 wv[RW][CPL];
#pragma unroll
  for (int r = 0; r < RW; ++r)
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
      const int c = lane + 64 * i;
      wv[r][i] = c < chunks ? *reinterpret_cast<const u32x4*>(wl + int64_t(j0 + r) * d + c * 8) : u32x4{0, 0, 0, 0};
    }
  float bj[RW];
#pragma unroll
  for (int r = 0; r < RW; ++r) bj[r] = __uint_as_float(uint32_t(p.bias[l][j0 + r]) << 16);
  float* ml = mod + int64_t(l) * n_seqs * rows;
  for (int b = 0; b < n_seqs; ++b) {
    const float* sr = s + int64_t(b) * d;
    float acc[RW];
#pragma unroll
    for (int r = 0; r < RW; ++r) acc[r] = 0.0f;
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
      const int c = lane + 64 * i;
      if (c < chunks) {
        const f32x4 lo = *reinterpret_cast<const f32x4*>(sr + c * 8);
        const f32x4 hi = *reinterpret_cast<const f32x4*>(sr + c * 8 + 4);
#pragma unroll
        for (int r = 0; r < RW; ++r)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            acc[r] += __uint_as_float(wv[r][i][e] << 16) * (e < 2 ? lo[2 * e] : hi[2 * e - 4]) +
                      __uint_as_float(wv[r][i][e] & 0xffff0000u) * (e < 2 ? lo[2 * e + 1] : hi[2 * e - 3]);
      }
    }
#pragma unroll
    for (int r = 0; r < RW; ++r) {
      const float v = wave_sum(acc[r]);
      if (lane == 0) ml[int64_t(b) * rows + j0 + r] = v + bj[r];
    }
  }
}

// One wave per row: y = fp16(((x - mean) / sqrt(var + eps)) * (1 + scale) + shift)
// with the row's sequence's scale and shift; fp32 statistics, the row kept in
// registers between the passes and the row's shift and scale loaded with it.
// CPL = 8-element chunks per lane (d <= 512 CPL).
template <typename TIn, int CPL>
__global__ __launch_bounds__(256) void ln_mod_kernel(const TIn* __restrict__ x, const float* __restrict__ mod,
                                                     const int32_t* __restrict__ row_seq, uint16_t* __restrict__ y,
                                                     int rows, int d, float eps, int shift_off, int scale_off) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int chunks = d >> 3;
  const float inv_d = 1.0f / float(d);
  for (int row = blockIdx.x * 4 + wave; row < rows; row += gridDim.x * 4) {
    const TIn* xr = x + int64_t(row) * d;
    const float* mrow = mod + int64_t(row_seq[row]) * (6 * d);
    float v[CPL][8];
    f32x4 sh[CPL][2], sc[CPL][2];
    float sum = 0.0f;
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
      const int c = lane + 64 * i;
      if (c < chunks) {
        if constexpr (sizeof(TIn) == 2) {
          const u32x4 u = *reinterpret_cast<const u32x4*>(xr + c * 8);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            v[i][2 * e] = __uint_as_float(u[e] << 16);
            v[i][2 * e + 1] = __uint_as_float(u[e] & 0xffff0000u);
          }
        } else {
          const f32x4 lo = *reinterpret_cast<const f32x4*>(xr + c * 8);
          const f32x4 hi = *reinterpret_cast<const f32x4*>(xr + c * 8 + 4);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            v[i][e] = lo[e];
            v[i][4 + e] = hi[e];
          }
        }
        sh[i][0] = *reinterpret_cast<const f32x4*>(mrow + shift_off + c * 8);
        sh[i][1] = *reinterpret_cast<const f32x4*>(mrow + shift_off + c * 8 + 4);
        sc[i][0] = *reinterpret_cast<const f32x4*>(mrow + scale_off + c * 8);
        sc[i][1] = *reinterpret_cast<const f32x4*>(mrow + scale_off + c * 8 + 4);
#pragma unroll
        for (int e = 0; e < 8; ++e) sum += v[i][e];
      }
    }
    const float mean = wave_sum(sum) * inv_d;
    float ss = 0.0f;
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
      const int c = lane + 64 * i;
      if (c < chunks) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          v[i][e] -= mean;
          ss += v[i][e] * v[i][e];
        }
      }
    }
    const float r = rsqrtf(wave_sum(ss) * inv_d + eps);
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
      const int c = lane + 64 * i;
      if (c < chunks) {
        float o[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          o[e] = v[i][e] * r * (1.0f + sc[i][0][e]) + sh[i][0][e];
          o[4 + e] = v[i][4 + e] * r * (1.0f + sc[i][1][e]) + sh[i][1][e];
        }
        u32x4 out;
#pragma unroll
        for (int e = 0; e < 4; ++e) out[e] = pack2h(o[2 * e], o[2 * e + 1]);
        *reinterpret_cast<u32x4*>(y + int64_t(row) * d + c * 8) = out;
      }
    }
  }
}

}  // namespace

hipError_t launch_silu_rows(const float* c, float* s, int n, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  const int grid = min((n + 255) / 256, 1024);
  hipLaunchKernelGGL(silu_rows_kernel, dim3(grid), dim3(256), 0, st, c, s, n);
  return hipGetLastError();
}

namespace {

template <int CPL, int RW>
hipError_t launch_mod(const DitModArgs& p, const float* s, float* mod, int n_seqs, int d, hipStream_t st) {
  const int64_t waves = (int64_t(p.n_layers) * 6 * d + RW - 1) / RW;
  hipLaunchKernelGGL((dit_mod_kernel<CPL, RW>), dim3(unsigned((waves + 3) / 4)), dim3(256), 0, st, p, s, mod, n_seqs,
                     d);
  return hipGetLastError();
}

template <typename TIn, int CPL>
hipError_t launch_ln(const TIn* x, const float* mod, const int32_t* row_seq, uint16_t* y, int rows, int d, float eps,
                     int shift_off, int scale_off, int grid, hipStream_t st) {
  hipLaunchKernelGGL((ln_mod_kernel<TIn, CPL>), dim3(grid), dim3(256), 0, st, x, mod, row_seq, y, rows, d, eps,
                     shift_off, scale_off);
  return hipGetLastError();
}

template <typename TIn>
hipError_t launch_ln_cpl(const TIn* x, const float* mod, const int32_t* row_seq, uint16_t* y, int rows, int d,
                         float eps, int shift_off, int scale_off, int grid, hipStream_t st) {
  const int cpl = (d / 8 + 63) / 64;
  if (cpl <= 1) return launch_ln<TIn, 1>(x, mod, row_seq, y, rows, d, eps, shift_off, scale_off, grid, st);
  if (cpl <= 2) return launch_ln<TIn, 2>(x, mod, row_seq, y, rows, d, eps, shift_off, scale_off, grid, st);
  if (cpl <= 4) return launch_ln<TIn, 4>(x, mod, row_seq, y, rows, d, eps, shift_off, scale_off, grid, st);
  if (cpl <= 8) return launch_ln<TIn, 8>(x, mod, row_seq, y, rows, d, eps, shift_off, scale_off, grid, st);
  return launch_ln<TIn, kMaxChunksPerLane>(x, mod, row_seq, y, rows, d, eps, shift_off, scale_off, grid, st);
}

}  // namespace

hipError_t launch_dit_modulation(const DitModArgs& p, const float* s, float* mod, int n_seqs, int d, hipStream_t st) {
  if (n_seqs <= 0 || p.n_layers <= 0) return hipSuccess;
  if (p.n_layers > kDitModLayers || d % 8 != 0 || d > 64 * kMaxChunksPerLane * 8) return hipErrorInvalidValue;
  const int cpl = (d / 8 + 63) / 64;
  // Rows per wave: about 8 KB of weights in flight per wave (RW divides 6 d
  // since d is a multiple of 8).
  if (cpl <= 1) return launch_mod<1, 8>(p, s, mod, n_seqs, d, st);
  if (cpl <= 2) return launch_mod<2, 4>(p, s, mod, n_seqs, d, st);
  if (cpl <= 4) return launch_mod<4, 2>(p, s, mod, n_seqs, d, st);
  if (cpl <= 8) return launch_mod<8, 1>(p, s, mod, n_seqs, d, st);
  return launch_mod<kMaxChunksPerLane, 1>(p, s, mod, n_seqs, d, st);
}

hipError_t launch_ln_modulate(const uint16_t* x, const float* x_f32, const float* mod, const int32_t* row_seq,
                              uint16_t* y, int rows, int d, float eps, int shift_off, int scale_off, int max_blocks,
                              hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  if (d % 8 != 0 || d > 64 * kMaxChunksPerLane * 8) return hipErrorInvalidValue;
  int grid = (rows + 3) / 4;
  if (max_blocks > 0 && grid > max_blocks) grid = max_blocks;
  if (x_f32) return launch_ln_cpl<float>(x_f32, mod, row_seq, y, rows, d, eps, shift_off, scale_off, grid, st);
  return launch_ln_cpl<uint16_t>(x, mod, row_seq, y, rows, d, eps, shift_off, scale_off, grid, st);
}

}  // namespace hs
