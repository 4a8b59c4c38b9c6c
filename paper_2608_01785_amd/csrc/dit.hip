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

// One wave per modulation row j: the row of W (bf16, d values) stays in
// registers while the wave takes its dot product with every sequence's
// silu(c).  mod[b][j] = bias[j] + sum_k s[b][k] W[j][k], fp32.
__global__ __launch_bounds__(256) void dit_mod_kernel(const uint16_t* __restrict__ w, const uint16_t* __restrict__ bias,
                                                      const float* __restrict__ s, float* __restrict__ mod,
                                                      int n_seqs, int d) {
  const int lane = threadIdx.x & 63;
  const int j = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int rows = 6 * d;
  if (j >= rows) return;
  const int chunks = d >> 3;
  float wv[kMaxChunksPerLane][8];
  const uint16_t* wr = w + int64_t(j) * d;
#pragma unroll
  for (int i = 0; i < kMaxChunksPerLane; ++i) {
    const int c = lane + 64 * i;
    if (c < chunks) {
      const u32x4 u = *reinterpret_cast<const u32x4*>(wr + c * 8);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        wv[i][2 * e] = __uint_as_float(u[e] << 16);
        wv[i][2 * e + 1] = __uint_as_float(u[e] & 0xffff0000u);
      }
    }
  }
  const float bj = __uint_as_float(uint32_t(bias[j]) << 16);
  for (int b = 0; b < n_seqs; ++b) {
    const float* sr = s + int64_t(b) * d;
    float acc = 0.0f;
#pragma unroll
    for (int i = 0; i < kMaxChunksPerLane; ++i) {
      const int c = lane + 64 * i;
      if (c < chunks) {
        const f32x4 lo = *reinterpret_cast<const f32x4*>(sr + c * 8);
        const f32x4 hi = *reinterpret_cast<const f32x4*>(sr + c * 8 + 4);
#pragma unroll
        for (int e = 0; e < 4; ++e) acc += wv[i][e] * lo[e] + wv[i][4 + e] * hi[e];
      }
    }
    acc = wave_sum(acc);
    if (lane == 0) mod[int64_t(b) * rows + j] = acc + bj;
  }
}

// One wave per row: y = fp16(((x - mean) / sqrt(var + eps)) * (1 + scale) + shift)
// with the row's sequence's scale and shift; fp32 statistics, the row kept in
// registers between the passes.
template <typename TIn>
__global__ __launch_bounds__(256) void ln_mod_kernel(const TIn* __restrict__ x, const float* __restrict__ mod,
                                                     const int32_t* __restrict__ row_seq, uint16_t* __restrict__ y,
                                                     int rows, int d, float eps, int shift_off, int scale_off) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int chunks = d >> 3;
  const float inv_d = 1.0f / float(d);
  for (int row = blockIdx.x * 4 + wave; row < rows; row += gridDim.x * 4) {
    const TIn* xr = x + int64_t(row) * d;
    float v[kMaxChunksPerLane][8];
    float sum = 0.0f;
#pragma unroll
    for (int i = 0; i < kMaxChunksPerLane; ++i) {
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
#pragma unroll
        for (int e = 0; e < 8; ++e) sum += v[i][e];
      }
    }
    const float mean = wave_sum(sum) * inv_d;
    float ss = 0.0f;
#pragma unroll
    for (int i = 0; i < kMaxChunksPerLane; ++i) {
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
    const float* mrow = mod + int64_t(row_seq[row]) * (6 * d);
#pragma unroll
    for (int i = 0; i < kMaxChunksPerLane; ++i) {
      const int c = lane + 64 * i;
      if (c < chunks) {
        const float* sh = mrow + shift_off + c * 8;
        const float* sc = mrow + scale_off + c * 8;
        const f32x4 sh0 = *reinterpret_cast<const f32x4*>(sh), sh1 = *reinterpret_cast<const f32x4*>(sh + 4);
        const f32x4 sc0 = *reinterpret_cast<const f32x4*>(sc), sc1 = *reinterpret_cast<const f32x4*>(sc + 4);
        float o[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          o[e] = v[i][e] * r * (1.0f + sc0[e]) + sh0[e];
          o[4 + e] = v[i][4 + e] * r * (1.0f + sc1[e]) + sh1[e];
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

hipError_t launch_dit_modulation(const uint16_t* w, const uint16_t* bias, const float* s, float* mod, int n_seqs,
                                 int d, hipStream_t st) {
  if (n_seqs <= 0) return hipSuccess;
  if (d % 8 != 0 || d > 64 * kMaxChunksPerLane * 8) return hipErrorInvalidValue;
  const int grid = (6 * d + 3) / 4;
  hipLaunchKernelGGL(dit_mod_kernel, dim3(grid), dim3(256), 0, st, w, bias, s, mod, n_seqs, d);
  return hipGetLastError();
}

hipError_t launch_ln_modulate(const uint16_t* x, const float* x_f32, const float* mod, const int32_t* row_seq,
                              uint16_t* y, int rows, int d, float eps, int shift_off, int scale_off, int max_blocks,
                              hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  if (d % 8 != 0 || d > 64 * kMaxChunksPerLane * 8) return hipErrorInvalidValue;
  int grid = (rows + 3) / 4;
  if (max_blocks > 0 && grid > max_blocks) grid = max_blocks;
  if (x_f32)
    hipLaunchKernelGGL(ln_mod_kernel<float>, dim3(grid), dim3(256), 0, st, x_f32, mod, row_seq, y, rows, d, eps,
                       shift_off, scale_off);
  else
    hipLaunchKernelGGL(ln_mod_kernel<uint16_t>, dim3(grid), dim3(256), 0, st, x, mod, row_seq, y, rows, d, eps,
                       shift_off, scale_off);
  return hipGetLastError();
}

}  // namespace hs
