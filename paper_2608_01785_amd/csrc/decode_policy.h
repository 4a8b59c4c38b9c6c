// Key-range split of single-row (decode) attention, shared by the planner and
// the kernels (constexpr, so usable on the device).  Pure C++; no HIP types.
#pragma once

#include <cstddef>
#include <cstdint>

namespace hs {

// Keys per tile (one wave's unit of work) and per split (one block: a tile
// per wave), by head size.
constexpr int dec_tile_keys(int dh) { return dh == 64 ? 64 : 32; }
constexpr int dec_split_keys(int dh) { return 4 * dec_tile_keys(dh); }
constexpr int dec_splits(int n_keys, int dh) { return (n_keys + dec_split_keys(dh) - 1) / dec_split_keys(dh); }

// Partial state of one split for one key/value head: G x dh unnormalised
// outputs, then G running maxima and G sums (floats, padded to 4).
constexpr int dec_part_floats(int group, int dh) { return (group * dh + 2 * group + 3) / 4 * 4; }

}  // namespace hs
