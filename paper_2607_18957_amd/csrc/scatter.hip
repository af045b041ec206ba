// Chunk -> tensor scatter for gfx950 (CDNA4), and the zero-fill used by the
// arena switch.
//
// The scatter is the device half of the refined tensor materialisation in
// InstantInfer (arXiv 2607.18957, Sec. 4.2): once a chunk is resident in
// device memory, every tensor piece it holds is copied into the tensor's own
// buffer ((C_i,InGPU)->(T_j,Alloc) moves T_j to Loaded). It is pure data
// movement, bound by HBM bandwidth: per payload byte one read of the chunk
// and one write of the tensor.
//
// Work split. One 128-thread workgroup (two wavefronts) owns one tile of
// tile_bytes (4 KiB by default), two 16-byte units per lane. Measured on a
// Llama-8B-shaped set against 256 threads x 8 KiB, 64 x 2 KiB, 8 and 16 KiB
// tiles, four or eight units per lane and persistent grids of 8 or 16
// workgroups per CU: two units per lane in small workgroups, one tile each,
// is fastest. The planner stores, per tile, the segment rows whose bytes
// meet it, so a workgroup reads only its own rows.
//   Ring (scatter_slot): a staged chunk's segment bytes are cut in segment
// order, gaps between segments skipped, so no workgroup exists for bytes no
// tensor needs (the gaps a sharded table leaves in the file). In a packed
// staging slot, and in a chunk without gaps, a tile's window is simply its
// share of the slot or chunk.
//   Resident image (scatter_layout): the tiles are windows of the plan's
// destination layout instead, the segments of all chunks in layout order.
// Each workgroup then writes one aligned 4 KiB block of destination memory
// (less any padding) and reads wherever its bytes lie. Writes that start or
// end inside a 128-byte line cost HBM bandwidth (a plain copy into a
// destination 48 bytes off a line runs 7% slower than an aligned one) while
// misaligned reads cost nothing measurable, so cutting by destination wins
// wherever source and destination offsets are not congruent modulo the
// tile (the 100,000-tensor set: 5.43 against 5.09 TB/s) and ties where
// they are (the Llama sets).
//
// Units. Destination memory is written in 16-byte blocks aligned to 16
// bytes, so every store of a block that a segment covers completely is one
// dwordx4 store. A unit is one (segment, destination block) pair. A unit
// belongs to the tile whose window holds its anchor: the coordinate of the
// first destination byte it covers -- its source offset in the chunk for
// the ring, its layout position for the resident image. Within a segment
// both coordinates grow with the destination address, so every unit has
// exactly one owner even when the source and destination phases (address
// mod 16) differ, and the units a tile owns are contiguous within each
// segment.
//
// Lanes to units. The workgroup stages its segment rows in LDS, counts each
// segment's units in the tile, and forms an exclusive prefix sum. Lane u of
// the tile's unit range then finds its segment by binary search over the
// prefix sums in LDS. Consecutive lanes get consecutive units, so a large
// segment is copied with fully coalesced 16-byte accesses, and many
// segments smaller than a wavefront (64 lanes x 16 B = 1 KiB) are served by
// one wavefront in the same pass. (The resident-image kernel's variant for
// tables of many small tensors skips this staging for tiles that one
// segment meets: every lane forms that one row itself.)
//
// Phase shift. The 16 source bytes of a destination block start at any
// address a. The lane loads the aligned 16-byte words at a & ~15 and
// (a & ~15) + 16 -- each only if it holds a byte the unit needs, so no load
// touches a 16-byte word outside the source data -- and assembles the block
// with funnel shifts (v_alignbit_b32). Blocks a segment covers only partly
// (its first and last block, or a segment shorter than 16 bytes) are
// written with 8/4/2/1-byte stores of exactly the covered bytes: padding and
// neighbouring tensors are never read-modify-written.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "scatter_math.h"
#include "scatter_types.h"

namespace ii {

static_assert((uint64_t)kMaxGridBlocks * kBlock <= 0xffffffffull,
              "one launch must stay within 2^32 - 1 work-items");
// scatter_slot launches the tiles of one chunk: at most 2^32 / 1024
static_assert((1ull << 32) / 1024 <= kMaxGridBlocks, "a chunk's tiles fit one launch");

namespace {

// Global-address-space accesses: plain pointers made from integer addresses
// would be generic (flat) accesses, which also count against the LDS wait
// counter.
#define II_GLOBAL __attribute__((address_space(1)))
typedef uint32_t v4u32 __attribute__((ext_vector_type(4)));
typedef II_GLOBAL v4u32 g_v4;
typedef II_GLOBAL uint64_t g_u64;
typedef II_GLOBAL uint32_t g_u32;
typedef II_GLOBAL uint16_t g_u16;
typedef II_GLOBAL uint8_t g_u8;

struct DevMem {
    __device__ __forceinline__ U4 ld16(uint64_t a) const {
        const v4u32 x = *reinterpret_cast<const g_v4*>(a);
        return U4{x.x, x.y, x.z, x.w};
    }
    // Whole destination blocks are streamed out with non-temporal stores: the
    // kernel never reads them back, and keeping them out of the caches leaves
    // room for the source stream (measured ~3% faster on large tables).
    __device__ __forceinline__ void st16(uint64_t a, U4 v) {
        v4u32 x = {v.x, v.y, v.z, v.w};
        __builtin_nontemporal_store(x, reinterpret_cast<g_v4*>(a));
    }
    __device__ __forceinline__ void st8(uint64_t a, uint32_t lo, uint32_t hi) {
        *reinterpret_cast<g_u64*>(a) = ((uint64_t)hi << 32) | lo;
    }
    __device__ __forceinline__ void st4(uint64_t a, uint32_t v) { *reinterpret_cast<g_u32*>(a) = v; }
    __device__ __forceinline__ void st2(uint64_t a, uint16_t v) { *reinterpret_cast<g_u16*>(a) = v; }
    __device__ __forceinline__ void st1(uint64_t a, uint8_t v) { *reinterpret_cast<g_u8*>(a) = v; }
};

// Inclusive prefix sum across the 64 lanes of a wavefront.
__device__ __forceinline__ uint32_t wave_scan(uint32_t v) {
    const uint32_t lane = threadIdx.x & 63u;
#pragma unroll
    for (uint32_t d = 1; d < 64; d <<= 1) {
        const uint32_t t = __shfl_up(v, d, 64);
        if (lane >= d) v += t;
    }
    return v;
}

}  // namespace

// Lane units base + j * kBlock + threadIdx.x (j < kUnroll) below total,
// row_at(u) giving the row of unit u; all stores follow all loads. Two issue
// orders:
//   kOverlap = false: each unit's phase shift follows its own loads, so the
//     wait for unit j's words comes before unit j + 1's loads issue -- at
//     most one unit's loads in flight per lane;
//   kOverlap = true: every unit's loads issue before any loaded word is
//     used, and all shifts precede the first store (a wait for loads issued
//     before a store would also wait for that store; the empty asm pins each
//     shifted block there, or the compiler sinks a unit's shift into its
//     store branch, after the previous unit's store).
// Measured: on tables of large tensors, where a tile is one unbroken 4 KiB
// stream, the first is faster (83.4% against 77.2% of HBM peak on a
// Llama-8B-shaped set); more loads in flight only lengthen the queues. On
// the 100,000-tensor set, whose tiles spend longer forming rows, the second
// is (68.1% against 65.7%).
template <bool kOverlap, class RowAt>
__device__ __forceinline__ void move_units(DevMem& mem, uint32_t base, uint32_t total,
                                           RowAt row_at) {
    UnitIO io[kUnroll];
    U4 v[kUnroll];
    if (kOverlap) {
        U4 x0[kUnroll], x1[kUnroll];
#pragma unroll
        for (int j = 0; j < kUnroll; ++j) {
            const uint32_t u = base + (uint32_t)j * kBlock + threadIdx.x;
            io[j].c0 = io[j].c1 = io[j].p = 0;  // every unit is shifted below
            x0[j] = x1[j] = U4{0, 0, 0, 0};
            if (u < total) {
                io[j] = unit_io(row_at(u), u);
                if (io[j].need0) x0[j] = mem.ld16(io[j].A);
                if (io[j].need1) x1[j] = mem.ld16(io[j].A + 16);
            }
        }
#pragma unroll
        for (int j = 0; j < kUnroll; ++j) {
            v[j] = funnel16(x0[j], x1[j], io[j].p);
            asm volatile("" : "+v"(v[j].x), "+v"(v[j].y), "+v"(v[j].z), "+v"(v[j].w));
        }
    } else {
#pragma unroll
        for (int j = 0; j < kUnroll; ++j) {
            const uint32_t u = base + (uint32_t)j * kBlock + threadIdx.x;
            io[j].c0 = io[j].c1 = 0;
            if (u < total) {
                io[j] = unit_io(row_at(u), u);
                U4 x0{0, 0, 0, 0}, x1{0, 0, 0, 0};
                if (io[j].need0) x0 = mem.ld16(io[j].A);
                if (io[j].need1) x1 = mem.ld16(io[j].A + 16);
                v[j] = funnel16(x0, x1, io[j].p);
            }
        }
    }
#pragma unroll
    for (int j = 0; j < kUnroll; ++j)
        if (io[j].c1 > io[j].c0) store_unit(mem, io[j].d, v[j], io[j].c0, io[j].c1);
}

// One workgroup's share of the scatter: the units anchored in its window,
// among segment rows [s_first, s_last). row(s, &cnt) returns the row of
// segment s seen from the window and its count of units anchored there.
// Every tile holds segment bytes, so s_first < s_last (the planner
// guarantees it); the batch loop runs at least once with no guard, which
// lets the argument loads issue together with the tile's own.
template <bool kOverlap, class RowOf>
__device__ __forceinline__ void scatter_tile(uint32_t s_first, uint32_t s_last, RowOf row) {
    __shared__ SegRow rows[kMaxSegBatch];
    __shared__ uint32_t pre[kMaxSegBatch];
    __shared__ uint32_t wsum[kBlock / 64];

    const uint32_t tid = threadIdx.x;
    DevMem mem;

    uint32_t s0 = s_first;
    do {
        const uint32_t ns = min((uint32_t)kMaxSegBatch, s_last - s0);
        uint32_t cnt = 0;
        if (tid < ns) rows[tid] = row(s0 + tid, &cnt);
        const uint32_t inc = wave_scan(cnt);
        if ((tid & 63u) == 63u) wsum[tid >> 6] = inc;
        __syncthreads();
        uint32_t before_wave = 0, total = 0;
#pragma unroll
        for (uint32_t w = 0; w < kBlock / 64; ++w) {
            const uint32_t x = wsum[w];
            before_wave += (w < (tid >> 6)) ? x : 0u;
            total += x;
        }
        if (tid < ns) {
            const uint32_t ex = before_wave + inc - cnt;
            pre[tid] = ex;
            rows[tid].ubase -= ex;
        }
        __syncthreads();

        for (uint32_t base = 0; base < total; base += kBlock * kUnroll)
            move_units<kOverlap>(mem, base, total,
                                 [&](uint32_t u) { return rows[find_row(pre, ns, u)]; });
        __syncthreads();  // rows/pre are rewritten by the next batch
        s0 += kMaxSegBatch;
    } while (s0 < s_last);
}

// Ring path: one chunk, staged in a device slot that starts at `slot`; one
// workgroup per tile of the chunk (`tiles` points at the chunk's first).
// implicit: tile m takes slot offsets [m * tile_bytes, ...) up to plen -- a
// packed slot, or a chunk without gaps at its own offsets; otherwise the
// slot holds a chunk with gaps at its own offsets and the tile's window of
// chunk offsets (`wins`, the chunk's first) applies.
__global__ __launch_bounds__(kBlock) void scatter_slot(
    const uint8_t* __restrict__ slot, const TileDev* __restrict__ tiles,
    const TileWin* __restrict__ wins, const SegDev* __restrict__ segs, uint32_t implicit,
    uint32_t tile_bytes, uint64_t plen) {
    const uint32_t g = blockIdx.x;
    const TileDev td = tiles[g];
    uint64_t w0, w1;
    if (implicit) {
        w0 = (uint64_t)g * tile_bytes;
        w1 = min(plen, w0 + tile_bytes);
    } else {
        const TileWin tw = wins[g];
        w0 = tw.w0;
        w1 = tw.w1;
    }
    const uint64_t cbase = reinterpret_cast<uint64_t>(slot);
    scatter_tile<false>(td.first, td.last, [&](uint32_t s, uint32_t* cnt) {
        const SegDev sd = segs[s];
        return make_row(sd.dst, sd.off, sd.len, cbase, w0, w1, cnt);
    });
}

// A tile that one segment meets, without LDS or barriers: every lane forms
// the row itself (its prefix is 0, so unit u is unit u of the row) -- the
// arithmetic of scatter_tile with a single row.
__device__ __forceinline__ void scatter_one_row(const SegRow& row, uint32_t total) {
    DevMem mem;
    for (uint32_t base = 0; base < total; base += kBlock * kUnroll)
        move_units<true>(mem, base, total, [&](uint32_t) { return row; });
}

// Resident-image path: the whole table in one dispatch (a grid of gy rows of
// gx workgroups, see grid_shape; tile g = y * gx + x, none past ntiles).
// `span` is the device address of the blob's span byte lo; segment rows are
// in layout order. Tile g takes the layout window w = win[g] (w = g when win
// is null: no window of the layout is all padding).
//   kMixed, chosen per plan (the planner's rule: enough tiles meet three or
// more segments): tiles that one segment meets skip the LDS staging and its
// barriers (scatter_one_row), and every tile issues all its loads before
// using any (move_units). Both put more loads in flight sooner, which pays
// where tiles spend long forming rows and costs on tables of large tensors
// (measured, 100,000-tensor set: 71.2% of HBM peak against 65.7%; a
// Llama-8B set: 77.2% against 83.4%; its rank-1-of-4 shard, whose tiles
// meet at most two segments: 76.2% against 80.0%).
template <bool kMixed>
__global__ __launch_bounds__(kBlock) void scatter_layout(
    const uint8_t* __restrict__ span, const TileDev* __restrict__ tiles,
    const uint32_t* __restrict__ win, const LayoutSeg* __restrict__ segs, uint32_t tile_bytes,
    uint32_t ntiles) {
    const uint32_t g = blockIdx.y * gridDim.x + blockIdx.x;
    if (g >= ntiles) return;
    const TileDev td = tiles[g];
    const uint64_t w0 = (uint64_t)(win ? win[g] : g) * tile_bytes;
    const uint64_t w1 = w0 + tile_bytes;
    const uint64_t sb = reinterpret_cast<uint64_t>(span);
    // source address of layout position x is sb + ls.src + (x - ls.pos)
    auto row_of = [&](uint32_t s, uint32_t* cnt) {
        const LayoutSeg ls = segs[s];
        return make_row(ls.dst, ls.pos, ls.len, sb + ls.src - ls.pos, w0, w1, cnt);
    };
    if (kMixed && td.last - td.first == 1) {
        uint32_t total;
        const SegRow row = row_of(td.first, &total);
        scatter_one_row(row, total);
        return;
    }
    scatter_tile<kMixed>(td.first, td.last, row_of);
}

// Zero the byte ranges [r.begin, r.end) (device addresses). One workgroup per
// range; 16-byte stores for whole aligned blocks, exact narrow stores at the
// edges.
__global__ __launch_bounds__(kBlock) void zero_ranges(const RangeDev* __restrict__ ranges,
                                                       uint32_t n) {
    if (blockIdx.x >= n) return;
    const RangeDev r = ranges[blockIdx.x];
    if (r.end <= r.begin) return;
    DevMem mem;
    const uint64_t b0 = r.begin >> 4, b1 = (r.end - 1) >> 4;
    const U4 z{0, 0, 0, 0};
    for (uint64_t b = b0 + threadIdx.x; b <= b1; b += kBlock) {
        const uint64_t d = b << 4;
        const uint64_t ds = d > r.begin ? d : r.begin;
        const uint64_t de = (d + 16) < r.end ? d + 16 : r.end;
        store_unit(mem, d, z, (uint32_t)(ds - d), (uint32_t)(de - d));
    }
}

hipError_t launch_scatter_slot(const uint8_t* slot, const TileDev* tiles, const TileWin* wins,
                               uint32_t ntiles, const SegDev* segs, bool implicit,
                               uint32_t tile_bytes, uint64_t plen, hipStream_t stream) {
    if (ntiles == 0) return hipSuccess;
    if (!implicit && !wins) return hipErrorInvalidValue;
    hipLaunchKernelGGL(scatter_slot, dim3(ntiles), dim3(kBlock), 0, stream, slot, tiles, wins,
                       segs, implicit ? 1u : 0u, tile_bytes, plen);
    return hipGetLastError();
}

hipError_t launch_scatter_layout(const uint8_t* span, const TileDev* tiles, const uint32_t* win,
                                 uint64_t ntiles, const LayoutSeg* segs, uint32_t tile_bytes,
                                 bool mixed, hipStream_t stream) {
    if (ntiles == 0) return hipSuccess;
    if (ntiles > 0x7fffffffull) return hipErrorInvalidConfiguration;
    uint32_t gx, gy;
    grid_shape(ntiles, &gx, &gy);
    if (mixed)
        hipLaunchKernelGGL(scatter_layout<true>, dim3(gx, gy), dim3(kBlock), 0, stream, span,
                           tiles, win, segs, tile_bytes, (uint32_t)ntiles);
    else
        hipLaunchKernelGGL(scatter_layout<false>, dim3(gx, gy), dim3(kBlock), 0, stream, span,
                           tiles, win, segs, tile_bytes, (uint32_t)ntiles);
    return hipGetLastError();
}

hipError_t launch_zero(const RangeDev* ranges, uint32_t n, hipStream_t stream) {
    for (uint32_t r0 = 0; r0 < n; r0 += kMaxGridBlocks) {
        const uint32_t m = std::min<uint32_t>(kMaxGridBlocks, n - r0);
        hipLaunchKernelGGL(zero_ranges, dim3(m), dim3(kBlock), 0, stream, ranges + r0, m);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace ii
