// The tables the scatter kernels read, as laid out in device memory. Shared
// by the kernels, the planner that builds them and the runtime that uploads
// them.
#pragma once

#include <cstdint>

namespace ii {

// One segment as the scatter kernel reads it: a piece of one tensor inside
// one chunk. 16 bytes so a wave loads its rows with dwordx4 loads.
struct SegDev {
    uint32_t off;  // offset of the piece inside its chunk
    uint32_t len;  // bytes
    uint64_t dst;  // device address the piece's first byte goes to
};
static_assert(sizeof(SegDev) == 16, "SegDev must stay 16 bytes");

// Work split of a chunk: tile m of a chunk takes the chunk's segment bytes
// [m * tile_bytes, (m+1) * tile_bytes) in segment order ("packed" offsets:
// a segment's bytes counted from the chunk's first segment, gaps between
// segments skipped). In a packed staging slot that is exactly the window
// [m * tile_bytes, ...) of the slot; in the chunk itself (a resident image,
// or a slot holding the chunk's bytes at their own offsets) the same bytes
// form the window [w0, w1) of chunk offsets. Either way the tile meets the
// segments [first, last). A chunk without segments has no tiles.
struct TileDev {
    uint32_t first;
    uint32_t last;
};
static_assert(sizeof(TileDev) == 8, "TileDev must stay 8 bytes");
// The tile's window [w0, w1) of chunk offsets, kept apart from TileDev so
// that launches whose windows follow from the tile index read only 8 bytes
// per tile.
struct TileWin {
    uint32_t w0;
    uint32_t w1;
};
static_assert(sizeof(TileWin) == 8, "TileWin must stay 8 bytes");

// One segment as the resident-image kernel reads it, in destination layout
// order: its bytes sit at span offset src (chunk * chunk_bytes + chunk
// offset) of the image and go to device address dst; pos is its layout
// position (the plan's destination offset of its first byte), the
// coordinate the image kernel's tiles are cut in. 32 bytes: two dwordx4
// loads per row.
struct LayoutSeg {
    uint64_t src;
    uint64_t dst;
    uint64_t pos;
    uint32_t len;
    uint32_t pad;
};
static_assert(sizeof(LayoutSeg) == 32, "LayoutSeg must stay 32 bytes");

// Zero-fill range for the switch scrub: [begin, end) as device addresses.
struct RangeDev {
    uint64_t begin;
    uint64_t end;
};

}  // namespace ii
