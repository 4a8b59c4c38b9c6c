// Skinny fp16 MFMA GEMM for decode-sized batches (M <= 128 rows), gfx950: one
// block per (weight strip, K split); the unit itself is in skinny_unit.h.
#include "skinny_unit.h"

namespace hs {
namespace {

using namespace skinny;

// NS: n-subtiles of 32 weight rows per block (1 or 2); MT: m-subtiles of 32
// rows.
template <int EPI, int DH, bool W_F16, int NS, int MT>
__global__ __launch_bounds__(kThreads) void skinny_kernel(GemmArgs a) {
  __shared__ __attribute__((aligned(1024))) uint8_t smem[SkinnyShape<NS, MT>::SMEM];
  skinny_unit<EPI, DH, W_F16, NS, MT>(a, blockIdx.x / a.n_split, blockIdx.x % a.n_split, smem);
}

template <int EPI, int DH, int NS, int MT>
hipError_t launch_mt(const GemmArgs& a, int n_blocks, hipStream_t s) {
  if (a.w_f16)
    hipLaunchKernelGGL((skinny_kernel<EPI, DH, true, NS, MT>), dim3(n_blocks), dim3(kThreads), 0, s, a);
  else
    hipLaunchKernelGGL((skinny_kernel<EPI, DH, false, NS, MT>), dim3(n_blocks), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

template <int EPI, int DH, int NS>
hipError_t launch_ns(const GemmArgs& a_in, int strips, hipStream_t s) {
  GemmArgs a = a_in;
  const int k_stages = a.K / BK;
  const SkinnySplit sp = skinny_split(strips, k_stages);
  a.n_split = (a.part && a.counters) ? sp.splits : 1;
  a.k_per_split = a.n_split > 1 ? sp.per : k_stages;
  const int n_blocks = strips * a.n_split;
  if (a.M <= 32) return launch_mt<EPI, DH, NS, 1>(a, n_blocks, s);
  if (a.M <= 64) return launch_mt<EPI, DH, NS, 2>(a, n_blocks, s);
  return launch_mt<EPI, DH, NS, 4>(a, n_blocks, s);
}

}  // namespace

bool skinny_supported(int epi, const GemmArgs& a) {
  if (a.M <= 0 || a.M > kSkinnyMaxRows || a.K % BK != 0) return false;
  if (epi == EPI_GATED || epi == EPI_GELU || (epi == EPI_QKV && !a.rope)) return false;  // large GEMM only
  if (epi == EPI_QKV) return a.dh == 64 || a.dh == 128;
  return true;
}

hipError_t launch_gemm_skinny(int epi, const GemmArgs& a, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  switch (epi) {
    case EPI_RESID: return launch_ns<EPI_RESID, 64, 1>(a, skinny_strips_resid(a.n_tiles_n * 256), s);
    case EPI_SWIGLU: return launch_ns<EPI_SWIGLU, 64, 2>(a, skinny_strips_swiglu(a.ffn), s);
    case EPI_QKV:
      return a.dh == 64 ? launch_ns<EPI_QKV, 64, 1>(a, skinny_strips_qkv(a.hq, a.hkv, 64), s)
                        : launch_ns<EPI_QKV, 128, 1>(a, skinny_strips_qkv(a.hq, a.hkv, 128), s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace hs
