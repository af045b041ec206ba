// Internal declarations shared by the planner and the runtime.
#pragma once

#include <algorithm>
#include <atomic>
#include <cstdint>
#include <memory>
#include <string>
#include <vector>

#include "ii.h"
#include "scatter_math.h"
#include "scatter_types.h"

namespace ii {

constexpr uint32_t kDefaultTile = 4u << 10;  // segment bytes per workgroup (<= kMaxTile)
constexpr uint32_t kMaxLanes = 4;             // streams a ring's chunks alternate between
constexpr uint64_t kIoAlign = 4096;           // block alignment of direct-I/O file reads
constexpr uint64_t kCopyAlign = 256;          // host-to-device copies start and end on these
constexpr uint32_t kMaxDmaGroups = 2;         // most copies a pinned chunk is moved with

// How a load from a pinned blob moves one chunk of a plan with gaps.
enum PinnedMove : uint8_t {
    kPinnedInPlace = 0,  // one copy of the used range, gaps included, at chunk offsets
    kPinnedGroups = 1,   // one 1-D or 2-D copy per run group, into the packed layout
    kPinnedGather = 2,   // host gather into the pinned slot, then one copy
};

// Runs of a chunk that share one length and one source distance between
// consecutive starts: count rows of len bytes, the first at chunk offset
// off, every stride bytes, landing back to back at packed offset poff --
// what one 2-D host-to-device copy moves (a single run has count 1).
struct DmaGroup {
    uint32_t off;
    uint32_t poff;
    uint32_t len;
    uint32_t count;
    uint32_t stride;
};

// A destination range [b, e) of tensor i (the destination checks).
struct DstRange {
    uint64_t b, e;
    size_t i;
};

// Static device workspace of ii_load_device_noalloc (runtime.hip).
constexpr uint64_t kScratchBytes = 64ull << 20;

struct Runtime;  // device-side state (runtime.hip)

void set_error(const char* fmt, ...);
int fail(int code, const char* fmt, ...);

}  // namespace ii

struct ii_plan_s {
    // table as given
    std::vector<std::string> names;
    std::vector<int32_t> dtype;
    std::vector<int32_t> ndim;
    std::vector<int64_t> shape_flat;
    std::vector<uint64_t> shape_start;
    std::vector<uint64_t> src_offset;
    std::vector<uint64_t> dst_align;
    std::vector<uint64_t> row_stride;  // 0 for contiguous tensors
    // derived
    std::vector<uint64_t> nbytes;
    std::vector<uint64_t> rows;        // 1 for contiguous tensors, 0 for empty ones
    std::vector<uint64_t> dst_offset;
    uint64_t payload = 0, arena_bytes = 0, max_align = 1;
    uint64_t lo = 0, hi = 0;
    uint64_t copy_bytes = 0;  // host-to-device bytes of a load from a pinned blob
    uint64_t chunk_bytes = 0;
    size_t num_chunks = 0;
    std::vector<uint64_t> chunk_seg_begin;  // num_chunks + 1
    // segments in chunk order, then by offset inside the chunk
    std::vector<uint32_t> seg_chunk, seg_off, seg_tensor, seg_len;
    std::vector<uint64_t> seg_toff;
    // Packed staging: when the host stage copies a chunk anyway (pageable
    // blob, file), it gathers only the segments' bytes, back to back in
    // segment order, so the link carries payload only. Segment s then sits
    // at seg_poff[s] of its slot; chunk k's slot holds chunk_plen[k] bytes.
    // A run is a maximal group of consecutive segments that are also
    // adjacent in the chunk (one memcpy): chunk offset run_off, slot offset
    // run_poff, run_len.
    bool packed_distinct = false;  // false: packed layout == chunk layout for every chunk
    // per chunk: how a load from a pinned blob moves it (PinnedMove) --
    // by copies of its run groups when it has at most kMaxDmaGroups of them,
    // else gathered on the host when more than a quarter of its used range
    // is gaps, else its used range in place
    std::vector<uint8_t> chunk_pinned;
    std::vector<uint64_t> chunk_group_begin;  // num_chunks + 1 (plans with gaps)
    std::vector<ii::DmaGroup> groups;
    std::vector<uint32_t> seg_poff;
    std::vector<uint64_t> chunk_plen;
    std::vector<uint64_t> chunk_run_begin;  // num_chunks + 1
    std::vector<uint32_t> run_off, run_poff, run_len;
    // ring tiles (see TileDev), chunk by chunk: what the scatter of one
    // staged or in-place chunk runs over
    uint32_t tile_bytes = ii::kDefaultTile;
    std::vector<ii::TileDev> tiles;
    std::vector<ii::TileWin> tile_win;       // plans with gaps only
    std::vector<uint64_t> chunk_tile_begin;  // num_chunks + 1
    // layout tiles (the resident-image kernel): the segments in destination
    // layout order -- lseg[j] is the j-th segment by layout position
    // dst_offset[tensor] + tensor offset -- and tiles of tile_bytes of
    // layout positions: tile g takes the window of layout positions
    // [w * tile_bytes, (w + 1) * tile_bytes) with w = lwin[g] (w = g when
    // lwin is empty: every window holds segment bytes) and the layout-order
    // segments [ltiles[g].first, ltiles[g].last) that meet it
    std::vector<uint32_t> lseg;
    std::vector<ii::TileDev> ltiles;
    std::vector<uint32_t> lwin;
    // whether the image kernel runs its variant for tables of many small
    // tensors (more loads in flight; see the planner's rule)
    bool layout_mixed = false;
    // host buffers of ii_load_device_noalloc, sized when the plan is made so
    // that the call itself allocates nothing: the layout-order segment rows
    // with resolved destinations, and the destination ranges its checks sort
    std::vector<ii::LayoutSeg> na_rows;
    std::vector<ii::DstRange> na_ranges;
    // runtime configuration
    uint32_t ring_depth = 3;
    uint32_t host_threads = 8;
    uint32_t copy_streams = 2;
    bool trace = false;
    // device state, created by the first load
    ii::Runtime* rt = nullptr;
    std::atomic<int> busy{0};

    uint64_t chunk_len(size_t k) const {
        return k + 1 < num_chunks ? chunk_bytes : (hi - lo) - chunk_bytes * (num_chunks - 1);
    }
    // The bytes of chunk k a load moves: from its first segment's start to
    // its last segment's end, rounded out to kCopyAlign inside the chunk;
    // empty if the chunk holds no segment (a gap between the tensors of a
    // sharded table).
    void chunk_used(size_t k, uint64_t* b, uint64_t* e) const {
        const uint64_t s0 = chunk_seg_begin[k], s1 = chunk_seg_begin[k + 1];
        if (s0 == s1) {
            *b = *e = 0;
            return;
        }
        const uint64_t a = ii::kCopyAlign;
        const uint64_t end = (uint64_t)seg_off[s1 - 1] + seg_len[s1 - 1];
        *b = seg_off[s0] & ~(a - 1);
        *e = std::min<uint64_t>(chunk_len(k), (end + a - 1) & ~(a - 1));
    }
};

namespace ii {
void runtime_destroy(ii_plan_t* p);
}
