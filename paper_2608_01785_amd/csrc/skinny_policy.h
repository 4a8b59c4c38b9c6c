// Work split of the skinny (decode-sized) GEMM, shared by the launcher and the
// workspace planner.  Pure C++; no HIP types.
#pragma once

#include <algorithm>
#include <cstddef>
#include <cstdint>

namespace hs {

constexpr int kSkinnyMaxRows = 128;      // M at or below this takes the skinny GEMM
constexpr int kSkinnyBK = 64;            // K per pipeline stage
constexpr int kSkinnyTargetBlocks = 128; // blocks wanted per launch
constexpr int kSkinnyMaxSplits = 8;
constexpr int kSkinnyMinStages = 8;      // K stages per split at least
constexpr int kSkinnySplitBelow = 128;   // only GEMMs with fewer strips split K ...
constexpr int kSkinnySplitFrom = 32;     // ... and only when K has this many stages
constexpr int kSkinnyMaxNormParts = 64;  // folded RMSNorm: partial sums per row a consumer prefetches

// 32-row activation subtiles covering M rows (1, 2 or 4).
inline int skinny_m_tiles(int M) { return M <= 32 ? 1 : (M <= 64 ? 2 : 4); }

// Activations of decode-sized batches are stored k-group-major with this many
// (padded) rows: element (m, k) at ((k / 8) * rows + m) * 8 + k % 8.  Rows
// M .. rows - 1 are never written; the GEMM discards their products.
inline int skinny_k8_rows(int M) { return 32 * skinny_m_tiles(M); }

struct SkinnySplit {
  int splits;  // blocks along K per weight strip
  int per;     // K stages per split (the last split may hold fewer)
};

// GEMMs with few weight strips split K until strips * splits reaches the
// target, keeping at least kSkinnyMinStages stages per split (a split's
// partial sums cost one extra round trip to memory) and no empty split.
inline SkinnySplit skinny_split(int strips, int k_stages) {
  if (strips >= kSkinnySplitBelow || k_stages < kSkinnySplitFrom) return {1, k_stages};
  int s = (kSkinnyTargetBlocks + strips - 1) / strips;
  s = std::min(s, kSkinnyMaxSplits);
  s = std::min(s, std::max(1, k_stages / kSkinnyMinStages));
  s = std::max(s, 1);
  const int per = (k_stages + s - 1) / s;
  s = (k_stages + per - 1) / per;
  return {s, per};
}

// Weight strips per GEMM: 32 output rows (residual GEMMs), 32 gate + 32 up
// rows (SwiGLU), 16 dimensions of one head and their RoPE partners (QKV).
inline int skinny_strips_resid(int n_out) { return n_out / 32; }
inline int skinny_strips_swiglu(int ffn) { return ffn / 32; }
inline int skinny_strips_qkv(int hq, int hkv, int dh) { return (hq + 2 * hkv) * (dh / 32); }

// fp32 partial sums of one split of one strip: NS x MT accumulator images of
// 16 registers x 64 lanes.
inline size_t skinny_partial_bytes(int ns, int m_tiles) { return size_t(ns) * m_tiles * 16 * 64 * 4; }

}  // namespace hs
