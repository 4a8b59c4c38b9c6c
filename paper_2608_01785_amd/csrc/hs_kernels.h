// Host-visible launch interface of the gfx950 kernels (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "decode_policy.h"
#include "skinny_policy.h"

namespace hs {

enum Epilogue : int {
  EPI_RESID = 1,   // out_f32 = resid + acc
  EPI_SWIGLU = 2,  // out = silu(gate) * up, gate/up rows gathered from [gate | up]
  EPI_QKV = 3,     // RoPE on Q and K heads, Q -> q buffer, K/V -> key/value store
  EPI_GATED = 4,   // out_f32 = resid + gate[seq(m)] * (acc + bias)   (large GEMM only)
  EPI_GELU = 5,    // out = gelu_tanh(acc + bias), fp16                  (large GEMM only)
};

struct GemmArgs {
  const uint16_t* A;  // activations [M, K] fp16: row-major, or k-group-major when k8_rows > 0
  const uint16_t* W;  // weights [N, K] row-major, bf16 (w_f16 = 0) or fp16 (w_f16 = 1)
  int w_f16;
  int M, K;
  int n_tiles_n;      // output tiles along N (256 weight rows each; 128 outputs for SWIGLU)
  uint16_t* out;      // SWIGLU output (fp16), row stride ldo, or k-group-major when k8_rows > 0
  float* out_f32;     // RESID output (fp32), row stride ldo
  int ldo;
  const uint16_t* resid;     // RESID: bf16 residual input with row stride ldo, or
  const float* resid_f32;    //        fp32 residual input (used when non-null)
  int ffn;                // SWIGLU: offset of the 'up' rows
  // QKV epilogue
  uint16_t* q;            // [M, hq, dh] fp16
  uint16_t* kstore;       // keys: element k_off[m] + g * kv_head_stride + d
  uint16_t* vstore;       // values: element v_off[m] + g * kv_head_stride + d * kv_tile_keys
  const int32_t* pos;     // RoPE positions: component c of row m at pos[c * pos_stride + m]
  int pos_stride;         // 0: one position per row
  int sec1, sec2;         // rotary pair j uses component (j >= sec1) + (j >= sec2)
  const int64_t* k_off;   // [M]
  const int64_t* v_off;   // [M]
  int64_t kv_head_stride; // elements between the heads of one slot (max_ctx * dh)
  const float2* rope;     // [max_pos, dh / 2] (cos, sin); null: no rotation (the large GEMM only)
  const uint16_t* bias;   // QKV: bf16 [(hq + 2 hkv) * dh] added before RoPE, or null; GATED / GELU: bf16 [N]
  const float* gate;      // GATED: row m scales by gate[row_seq[m] * gate_stride + n]
  int gate_stride;
  const int32_t* row_seq; // GATED: sequence of each row
  int hq, hkv, dh;
  // Skinny GEMM split along K: fp32 partial sums and one arrival counter per
  // weight strip (zero on entry, left at zero on exit).
  float* part;
  int32_t* counters;
  int n_split, k_per_split;  // set by the launcher
  // RMSNorm folded into the skinny GEMMs around it.  RESID, optional: the
  // new residual's per-row partial sums of squares over each 32-column strip
  // (sumsq_out[m * strips + strip]) and the residual times a per-column gain
  // in fp16 (scaled_out, row stride ldo).
  float* sumsq_out;
  uint16_t* scaled_out;      // row stride ldo, or k-group-major when k8_rows > 0
  const uint16_t* gain;      // bf16 [ldo]
  // QKV / SWIGLU, optional: row m of the product is multiplied by
  // rsqrt(sum_p row_sumsq[m * row_parts + p] / K + eps) before RoPE or SiLU
  // (row_parts a multiple of 4, at most kSkinnyMaxNormParts).
  const float* row_sumsq;
  int row_parts;
  float eps;
  // Skinny GEMM only: A, out and scaled_out are k-group-major with this many
  // padded rows (skinny_k8_rows(M)); 0 = row-major.
  int k8_rows;
  // Timing mode: four counters of the launch (see LaunchClock), or null.
  uint64_t* clock;
};

// The large GEMM does not take the folded-RMSNorm fields (they must be null).
hipError_t launch_gemm(int epi, const GemmArgs& a, int max_blocks, hipStream_t s);

// Decode-sized GEMMs (M <= kSkinnyMaxRows): thin weight strips, K split
// across blocks as skinny_split() says.
bool skinny_supported(int epi, const GemmArgs& a);
hipError_t launch_gemm_skinny(int epi, const GemmArgs& a, hipStream_t s);

struct AttnArgs {
  const uint16_t* q;        // [T, hq, dh]
  const uint16_t* kstore;   // keys, layout as the cache (kv_tile_keys)
  const uint16_t* vstore;   // values in transposed tiles, layout as the cache
  uint16_t* o;              // [T, hq * dh], k-group-major when o_k8_rows > 0
  int o_k8_rows;
  const int32_t* items;     // [n_items][2] = (sequence, first query row within it)
  int n_items;
  const int32_t* seq_start; // [B] first packed row
  const int32_t* seq_len;   // [B] query rows
  const int32_t* seq_ctx;   // [B] cached rows before the chunk
  const int32_t* seq_page0; // [B] index of the sequence's first page in page_base
  const int64_t* page_base; // element offset of a page's position 0 (head 0, dim 0); keys and values alike
  int page_keys;            // positions per page, a multiple of 64 (one key tile never straddles pages)
  int64_t kv_head_stride;
  int hq, hkv, dh;
  float scale_log2;         // log2(e) / sqrt(dh)
  int bidirectional;        // 0: causal (bottom-right); 1: every row sees every key of its sequence
  uint64_t* clock;          // timing mode: four counters of the launch (see LaunchClock), or null
};

hipError_t launch_attention(const AttnArgs& a, hipStream_t s);

// Single-row (decode) attention: one block per (work item, key/value head);
// a work item is one key range (unit_keys keys, inside one page) of one row
// and carries everything the block needs, so the K/V loads follow a single
// record load.
struct DecItem {
  int32_t t;        // packed row of the query
  int32_t n_keys;   // keys the row attends to (cached prefix + itself)
  int32_t split;    // key range split * unit_keys ..
  int32_t n_split;  // splits of this row (its items are consecutive)
  int64_t kbase;    // element offset of position 0 (head 0) of the page holding the range
  int64_t vbase;    // the same for values (dim 0)
};
static_assert(sizeof(DecItem) == 32, "decode item record");

struct DecodeAttnArgs {
  const uint16_t* q;
  const uint16_t* kstore;   // keys, layout as the cache (kv_tile_keys)
  const uint16_t* vstore;   // values in transposed tiles, layout as the cache
  uint16_t* o;               // [T, hq * dh], k-group-major when o_k8_rows > 0
  int o_k8_rows;
  const DecItem* items;
  int n_items;              // work items the grid covers
  const int32_t* n_items_dev;  // or null; else the call's items on the device (<= n_items), the rest exit
  float* part;              // [n_items][hkv][dec_part_floats] partial states of split rows
  int32_t* counters;        // [n_items * hkv] arrival counters (first item of a row), zero on entry and exit
  int64_t kv_head_stride;
  int page_keys;            // positions per page (the key range's page starts at split * unit_keys rounded down)
  int unit_keys;            // keys per work item: divides dec_split_keys(dh), and page_keys on a paged cache
  int hq, hkv, dh;
  float scale_log2;
};

hipError_t launch_decode_attention(const DecodeAttnArgs& a, hipStream_t s);

// x is bf16 (x_f32 null) or fp32 (x_f32 non-null); y is fp16, row-major or
// k-group-major with k8_rows padded rows (k8_rows > 0).
hipError_t launch_rmsnorm(const uint16_t* x, const float* x_f32, const uint16_t* gamma, uint16_t* y, int rows,
                          int d, float eps, int k8_rows, int max_blocks, hipStream_t s);

hipError_t launch_rope_table(float2* tab, int max_pos, int dh, float base, hipStream_t s);

// Diffusion-transformer pieces (dit.hip).  s = silu(c) for B x d conditioning
// values (fp32); for each of n_layers (at most kDitModLayers) layers l,
// mod[l][b][j] = bias_l[j] + sum_k s[b][k] W_l[j][k] over its 6d modulation
// rows (W_l bf16 [6d, d] row-major, bias_l bf16 [6d]).
constexpr int kDitModLayers = 8;
struct DitModArgs {
  const uint16_t* w[kDitModLayers];
  const uint16_t* bias[kDitModLayers];
  int n_layers;
};
hipError_t launch_silu_rows(const float* c, float* s, int n, hipStream_t st);
hipError_t launch_dit_modulation(const DitModArgs& p, const float* s, float* mod, int n_seqs, int d, hipStream_t st);
// y[t] = fp16(LN(x[t]) * (1 + mod[b][scale_off + j]) + mod[b][shift_off + j]),
// b = row_seq[t]; x bf16 (x_f32 null) or fp32; mod rows of 6d floats.
hipError_t launch_ln_modulate(const uint16_t* x, const float* x_f32, const float* mod, const int32_t* row_seq,
                              uint16_t* y, int rows, int d, float eps, int shift_off, int scale_off, int max_blocks,
                              hipStream_t st);

hipError_t launch_probe(uint32_t* out, int n_groups, hipStream_t s);

// dst = fp16(src) for n bf16 values (n even).
// Static device scratch of the no-allocation decode step (noalloc.hip): its
// size, and its address on `device`, which must be the current device on the
// first call for it (later calls return the kept address).
size_t noalloc_scratch_bytes();
constexpr int kNoAllocMaxBatch = 1024;  // rows of one no-allocation decode step
hipError_t noalloc_scratch_resolve(int device, void** out);

hipError_t launch_convert_bf16_f16(const uint16_t* src, uint16_t* dst, int64_t rows, int64_t cols, hipStream_t s);

}  // namespace hs
