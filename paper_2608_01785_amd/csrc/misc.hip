// RMSNorm, RoPE table and topology-probe kernels for gfx950.
#include "hs_device.h"
#include "hs_kernels.h"

namespace hs {
namespace {

constexpr int kMaxChunksPerLane = 16;  // hidden <= 64 lanes * 16 chunks * 8 = 8192

// One wave per row: y = x / sqrt(mean(x^2) + eps) * gamma, fp32 reduction,
// fp16 output (the next GEMM's operand).  The input row (bf16 or fp32) stays in registers between the
// two passes; loads are 16 bytes wide.
// CPL = 8-element chunks per lane (d <= 512 CPL): registers for the row only.
template <typename TIn, int CPL>
__global__ __launch_bounds__(256) void rmsnorm_kernel(const TIn* __restrict__ x, const uint16_t* __restrict__ gamma,
                                                      uint16_t* __restrict__ y, int rows, int d, float eps,
                                                      int k8_rows) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int chunks = d >> 3;  // 8 elements per chunk
  const float inv_d = 1.0f / float(d);
  for (int row = blockIdx.x * 4 + wave; row < rows; row += gridDim.x * 4) {
    const TIn* xr = x + int64_t(row) * d;
    float v[CPL][8];
    float ss = 0.0f;
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
#pragma unroll
        for (int e = 0; e < 8; ++e) ss += v[i][e] * v[i][e];
      }
    }
    ss = wave_sum(ss);
    const float r = rsqrtf(ss * inv_d + eps);
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
      const int c = lane + 64 * i;
      if (c < chunks) {
        const u32x4 gv = *reinterpret_cast<const u32x4*>(gamma + c * 8);
        u32x4 out;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float lo = v[i][2 * e] * r * __uint_as_float(gv[e] << 16);
          const float hi = v[i][2 * e + 1] * r * __uint_as_float(gv[e] & 0xffff0000u);
          out[e] = pack2h(lo, hi);
        }
        *reinterpret_cast<u32x4*>(y + act_index(row, c * 8, d, k8_rows)) = out;
      }
    }
  }
}

// tab[p, j] = (cos, sin)(p * base^(-2j/dh)), angle formed in double precision.
__global__ void rope_table_kernel(float2* tab, int max_pos, int dh, double base) {
  const int half = dh / 2;
  const int64_t n = int64_t(max_pos) * half;
  for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += int64_t(gridDim.x) * blockDim.x) {
    const int p = int(i / half), j = int(i % half);
    const double inv = pow(base, -2.0 * double(j) / double(dh));
    double s, c;
    sincos(double(p) * inv, &s, &c);
    tab[i] = make_float2(float(c), float(s));
  }
}

// HW_ID (hardware register 4) and XCC_ID (hardware register 20), full 32 bits.
constexpr int kHwRegHwId = (31 << 11) | 4;
constexpr int kHwRegXccId = (31 << 11) | 20;

// Each block records where it ran: XCC id, shader engine, CU (shader-array
// bit and CU id), and the constant 100 MHz clock.  Blocks then wait about
// 20 microseconds (bounded) so that the dispatcher spreads them over CUs.
__global__ void probe_kernel(uint32_t* out, int n) {
  if (threadIdx.x == 0 && blockIdx.x < n) {
    const uint32_t hw = __builtin_amdgcn_s_getreg(kHwRegHwId);
    const uint32_t xcc = __builtin_amdgcn_s_getreg(kHwRegXccId);
    const uint64_t t0 = wall_clock64();
    u32x4 rec;
    rec.x = xcc & 0xfu;
    rec.y = (hw >> 13) & 0x7u;
    rec.z = (((hw >> 12) & 1u) << 4) | ((hw >> 8) & 0xfu);
    rec.w = uint32_t(t0);
    *reinterpret_cast<u32x4*>(out + 4 * int64_t(blockIdx.x)) = rec;
    while (wall_clock64() - t0 < 2000) {
    }
  }
}

// Weight preparation: pairs of bf16 values -> pairs of fp16 values.
// bf16 [rows, cols] row-major -> fp16 panel-major [cols / 32][rows][32], two
// elements per thread.
__global__ void convert_kernel(const uint32_t* __restrict__ src, uint32_t* __restrict__ dst, int64_t rows,
                               int64_t cols) {
  const int64_t n2 = rows * cols / 2, half_cols = cols / 2;
  for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n2; i += int64_t(gridDim.x) * blockDim.x) {
    const int64_t r = i / half_cols, c = 2 * (i % half_cols);
    dst[(((c >> 5) * rows + r) * 32 + (c & 31)) >> 1] = bf2x_to_h2x(src[i]);
  }
}

}  // namespace

hipError_t launch_convert_bf16_f16(const uint16_t* src, uint16_t* dst, int64_t rows, int64_t cols, hipStream_t s) {
  const int64_t n2 = rows * cols / 2;
  if (n2 <= 0) return hipSuccess;
  int64_t grid = (n2 + 255) / 256;
  if (grid > 8192) grid = 8192;
  hipLaunchKernelGGL(convert_kernel, dim3(unsigned(grid)), dim3(256), 0, s, reinterpret_cast<const uint32_t*>(src),
                     reinterpret_cast<uint32_t*>(dst), rows, cols);
  return hipGetLastError();
}

namespace {

template <typename TIn, int CPL>
hipError_t launch_norm(const TIn* x, const uint16_t* gamma, uint16_t* y, int rows, int d, float eps, int k8_rows,
                       int grid, hipStream_t s) {
  hipLaunchKernelGGL((rmsnorm_kernel<TIn, CPL>), dim3(grid), dim3(256), 0, s, x, gamma, y, rows, d, eps, k8_rows);
  return hipGetLastError();
}

// The instance for exactly cpl chunks per lane (1 .. kMaxChunksPerLane).
template <typename TIn, int CPL = 1>
hipError_t launch_norm_cpl(int cpl, const TIn* x, const uint16_t* gamma, uint16_t* y, int rows, int d, float eps,
                           int k8_rows, int grid, hipStream_t s) {
  if constexpr (CPL < kMaxChunksPerLane) {
    if (cpl > CPL) return launch_norm_cpl<TIn, CPL + 1>(cpl, x, gamma, y, rows, d, eps, k8_rows, grid, s);
  }
  return launch_norm<TIn, CPL>(x, gamma, y, rows, d, eps, k8_rows, grid, s);
}

}  // namespace

hipError_t launch_rmsnorm(const uint16_t* x, const float* x_f32, const uint16_t* gamma, uint16_t* y, int rows,
                          int d, float eps, int k8_rows, int max_blocks, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  int grid = (rows + 3) / 4;
  if (grid > max_blocks) grid = max_blocks;
  const int cpl = (d / 8 + 63) / 64;  // 1 .. kMaxChunksPerLane
  if (x_f32) return launch_norm_cpl<float>(cpl, x_f32, gamma, y, rows, d, eps, k8_rows, grid, s);
  return launch_norm_cpl<uint16_t>(cpl, x, gamma, y, rows, d, eps, k8_rows, grid, s);
}

hipError_t launch_rope_table(float2* tab, int max_pos, int dh, float base, hipStream_t s) {
  if (max_pos <= 0) return hipSuccess;
  const int64_t n = int64_t(max_pos) * (dh / 2);
  int grid = int((n + 255) / 256);
  if (grid > 4096) grid = 4096;
  hipLaunchKernelGGL(rope_table_kernel, dim3(grid), dim3(256), 0, s, tab, max_pos, dh, double(base));
  return hipGetLastError();
}

hipError_t launch_probe(uint32_t* out, int n_groups, hipStream_t s) {
  if (n_groups <= 0) return hipSuccess;
  hipLaunchKernelGGL(probe_kernel, dim3(n_groups), dim3(64), 0, s, out, n_groups);
  return hipGetLastError();
}

}  // namespace hs
