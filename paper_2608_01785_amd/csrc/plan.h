// Host-only planner: validation, batch metadata, work lists and workspace
// layout.  Pure C++ (no HIP), so it builds with g++ for sanitizer runs.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "horizon.h"

namespace hs {

void set_error(const char* fmt, ...);
hs_status fail(hs_status s, const char* fmt, ...);
void clear_error();

constexpr int kMaxXcc = 8;
constexpr size_t kAlign = 256;
constexpr int kAttnBlockQ = 128;   // query rows per prefill-attention block

inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

hs_status validate_cfg(const hs_layer_cfg* cfg);

// Checks offsets (and optional cached lengths); returns T and the largest
// position + 1 over all rows.
hs_status validate_batch(const int32_t* seq_offsets, const int32_t* ctx_lens, int32_t n_seqs,
                         int32_t* n_tokens, int32_t* max_pos);

// The GEMMs address activations and weights through buffer resources whose
// size and offsets are 32-bit byte counts, and single-row attention addresses
// a cache page the same way within 2 GiB.  HS_ERR_UNSUPPORTED when a layer's
// weight matrix, an activation matrix of T rows, or a cache page of max_ctx
// positions (0: no cache) would not fit.
hs_status check_32bit_extents(const hs_layer_cfg& cfg, int32_t n_tokens, int32_t max_ctx);

// Byte offsets of every buffer inside the caller's workspace.
struct WsLayout {
  size_t meta;        // metadata image (copied from the host each call)
  size_t meta_bytes;
  size_t n;           // [T, d] normalised rows
  size_t q;           // [T, hq, dh]
  size_t kpack;       // keys when no cache is given: one slot of packed_ctx positions
  size_t vpack;       // values when no cache is given, same
  int64_t packed_ctx; // positions of that slot: every sequence starts 64-aligned, plus 64
  size_t o;           // [T, hq * dh]
  size_t h;           // [T, d] fp32 residual after attention
  size_t a;           // [T, ffn]
  size_t xtmp;        // [T, d] fp32 residual between layers
  size_t sumsq;       // [T, d / 32] fp32 partial sums of squares of the residual (folded RMSNorm)
  size_t rope;        // [max_pos, dh / 2] float2
  size_t part;        // split-K partial sums of the skinny GEMM (T <= 128 rows only)
  size_t part_bytes;
  size_t dec_part;    // per-split partial states of single-row attention
  size_t dec_part_bytes;
  size_t total;
};

// Upper bounds used for sizing: T rows, B sequences, positions < max_pos.
int64_t max_att_items(int32_t T, int32_t B);

// page_keys: positions per page of a paged cache, 0 without a block table.
// packs: reserve the packed key/value slot that calls without a cache use
// (false only for a call that is known to carry a cache).
WsLayout ws_layout(const hs_layer_cfg& c, int32_t T, int32_t B, int32_t max_pos, int32_t page_keys = 0,
                   bool packs = true);

// Keys per single-row attention work unit: the head size's split, cut down
// to a divisor of the page size on a paged cache so that no unit straddles
// two pages.
int32_t dec_unit_keys(int dh, int32_t page_keys);

// Metadata of one call, laid out as one host image mirrored in the workspace.
struct Plan {
  int32_t T = 0, B = 0, max_pos = 0;
  std::vector<uint8_t> image;
  // byte offsets inside image
  size_t pos = 0, k_off = 0, v_off = 0;
  size_t pos3 = 0;  // [3][T] multimodal RoPE positions (filled only when given)
  size_t row_seq = 0;  // [T] int32: sequence of each packed row
  size_t seq_start = 0, seq_len = 0, seq_ctx = 0;
  size_t seq_page0 = 0;  // [B] int32: index of the sequence's first page in page_base
  size_t page_base = 0;  // [n_pages] int64: element offset of a page's position 0, head 0
  int32_t n_pages = 0;
  int32_t page_keys = 0;  // positions per page (a slot, or the packed buffer, is one page)
  int32_t unit_keys = 0;  // keys per single-row attention work unit
  size_t att_items = 0, dec_rows = 0;
  size_t counters = 0;  // split-K arrival counters of the skinny GEMM, zero in the image
  size_t dec_items = 0;  // [n_dec_items] 32-byte records (row, keys, split, splits, K base, V base)
  size_t dec_count = 0;  // [n_dec_items * hkv] arrival counters, zero in the image
  int32_t n_att_items = 0, n_dec_rows = 0, n_counters = 0, n_dec_items = 0;
  size_t dec_n = 0;      // int32: n_dec_items, for kernels launched with a grid for the capacity
  int64_t cap_dec_items = 0;  // decode work items the layout holds (== n_dec_items unless fixed)
  int64_t kv_head_stride = 0;
};

// A fixed layout: every region of the image sized for the largest batch of
// this shape whose positions stay below max_pos (the bounds the workspace
// layout reserves), so that region offsets, the image size and the single-row
// attention grid do not depend on the call's lengths.  Kernels replayed from
// a captured graph read the call's metadata from such an image.
struct PlanCapacity {
  int32_t max_pos = 0;
  int32_t page_keys = 0;  // positions per page of a paged cache, 0 without a block table
};

// Key/value placement: packed (no cache, rows in the workspace), cache slots
// (sequence b in slot b) or pages named by a block table.
struct KvPlacement {
  bool cache = false;
  int32_t max_ctx = 0;             // positions per slot (per page with a table)
  int64_t packed_ctx = 0;
  const int32_t* table = nullptr;  // host [B][pages_per_seq] slot indices, or null
  int32_t pages_per_seq = 0;
};

// Checks a block table against a batch: every page a sequence reaches names
// a slot in [0, n_slots), no sequence lists a page twice among the pages it
// reaches, and a page that receives new rows is reached by no other sequence.
hs_status check_block_table(const int32_t* table, int32_t pages_per_seq, int32_t n_slots, int32_t page_keys,
                            const int32_t* seq_offsets, const int32_t* ctx_lens, int32_t n_seqs);

hs_status build_plan(const hs_layer_cfg& c, const int32_t* seq_offsets, const int32_t* ctx_lens,
                     int32_t n_seqs, const KvPlacement& kv, Plan* out, const int32_t* positions3 = nullptr,
                     const PlanCapacity* cap = nullptr, bool bidirectional = false);

}  // namespace hs
