// Key-range split of single-row (decode) attention, shared by the planner and
// the kernels (constexpr, so usable on the device).  Pure C++; no HIP types.
#pragma once

#include <cstddef>
#include <cstdint>

namespace hs {

// Keys per tile (a wave's step: 32 keys, 8 or 16 KB of keys and values) and
// per split (one block; its four waves take every fourth tile), by head size.
constexpr int dec_tile_keys(int dh) { return dh == 64 ? 32 : 32; }
constexpr int dec_split_keys(int dh) { return dh == 64 ? 1024 : 512; }
constexpr int dec_splits(int n_keys, int dh) { return (n_keys + dec_split_keys(dh) - 1) / dec_split_keys(dh); }

// Key/value cache layout, per layer (elements are fp16):
//   K: [slot][Hkv][max_ctx][dh]                        key rows of a head contiguous
//   V: [slot][Hkv][max_ctx / kv_tile_keys][dh][kv_tile_keys]
//      values transposed in tiles of kv_tile_keys keys, so a tile of one
//      head is one contiguous 4 or 8 KB block
// Both hold max_ctx * dh elements per (slot, head).  max_ctx is a multiple
// of 64.
constexpr int kv_tile_keys = 32;

// Partial state of one split for one key/value head: G x dh unnormalised
// outputs, then G running maxima and G sums (floats, padded to 4).
constexpr int dec_part_floats(int group, int dh) { return (group * dh + 2 * group + 3) / 4 * 4; }

}  // namespace hs
