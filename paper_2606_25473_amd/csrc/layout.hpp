// layout.hpp -- host-side mask handling (C++17, no HIP dependency).
#pragma once

#include <stdint.h>

#include <string>

#include "attn_jvp.h"
#include "schedule.hpp"

namespace attn {

// Validate `layout` against the sequence length L and derive its query-group
// table (ranges of each group sorted, empty ones dropped, touching ones merged).
// Returns false and fills *err on an invalid layout.
bool build_groups(const attn_chunk_layout* layout, int L, GroupTable* gt, std::string* err);

// Admissible (query, key) pairs of the mask, one (batch, head).
int64_t count_pairs(const GroupTable& gt);

// Pairs evaluated by a kernel with br-row query tiles and bc-key blocks.
int64_t count_computed_pairs(const GroupTable& gt, int L, int br, int bc);

// Work-group -> query-tile order for the layout (heaviest tiles first).
TileOrder make_tile_order(const attn_chunk_layout* layout, int L, int br);

// Tile order when the rows below t0 carry no tangent (their tiles need the primal
// only): the tiles wholly below t0 and the others, each heaviest first, merged by
// estimated cost (mode 3; mode 2 beyond kMaxMergeTiles tiles).
TileOrder make_tile_order_zero_clean(const GroupTable& gt, int L, int br, int bc, int t0);

}  // namespace attn
