// Merge planner: tensor table -> chunks, segments, destination layout, tiles.
//
// Sec. 4.2 ("Refined CFA Model") of InstantInfer (arXiv 2607.18957) divides
// the model file into equal-length chunks, the last possibly partial, and
// precomputes which tensors each chunk holds and which chunks each tensor
// spans. This file computes that association once, on the host, so that the
// load path only walks precomputed tables.
//
// Method: list every non-empty tensor's source pieces -- the tensor itself,
// or each of its rows when it is given with a row stride (a tensor-parallel
// shard read out of an unsharded file) -- sort them by source offset (which
// also finds overlaps), then sweep them in source order and cut each piece at
// chunk boundaries. Because pieces are disjoint, the segments come out
// already ordered by chunk and by offset inside the chunk: O(P log P + S) for
// P pieces. The per-tile segment windows used by the kernel come from one
// more linear sweep per chunk.
#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <new>
#include <unistd.h>

#include "ii_internal.h"

namespace ii {

static thread_local std::string g_last_error;

void set_error(const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
}

int fail(int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return code;
}

static int width_of(int32_t dtype) {
    switch (dtype) {
    case II_U8: case II_I8: case II_FP8_E4M3: case II_FP8_E5M2: return 1;
    case II_BF16: case II_F16: return 2;
    case II_F32: case II_I32: return 4;
    case II_F64: case II_I64: return 8;
    default: return 0;
    }
}

static bool pow2(uint64_t x) { return x && !(x & (x - 1)); }

// One contiguous run of a tensor's source bytes: the whole tensor, or one
// row of a tensor given with a row stride.
struct Piece {
    uint64_t src;   // blob offset of the first byte
    uint64_t len;
    uint64_t toff;  // offset of that byte inside the tensor
    uint32_t tensor;
};

static uint32_t env_u32(const char* name, uint32_t dflt, uint32_t lo, uint32_t hi) {
    const char* s = getenv(name);
    if (!s || !*s) return dflt;
    char* end = nullptr;
    unsigned long v = strtoul(s, &end, 10);
    if (end == s || v < lo || v > hi) return dflt;
    return (uint32_t)v;
}

}  // namespace ii

using namespace ii;

extern "C" int ii_plan(const ii_tensor_desc* table, size_t n, uint64_t chunk_bytes,
                       ii_plan_t** out) {
    if (!out) return fail(II_EINVAL, "ii_plan: out is NULL");
    *out = nullptr;
    if (n && !table) return fail(II_EINVAL, "ii_plan: table is NULL");
    if (chunk_bytes < 16 || chunk_bytes % 16 || chunk_bytes >= (1ull << 32))
        return fail(II_EINVAL, "ii_plan: chunk_bytes %llu must be a multiple of 16 in [16, 2^32)",
                    (unsigned long long)chunk_bytes);
    if (n >= (1ull << 32) - 1) return fail(II_EINVAL, "ii_plan: too many tensors");

    std::unique_ptr<ii_plan_t> p;
    try {
        p.reset(new ii_plan_t());
        p->names.resize(n);
        p->dtype.resize(n);
        p->ndim.resize(n);
        p->shape_start.resize(n);
        p->src_offset.resize(n);
        p->dst_align.resize(n);
        p->row_stride.resize(n);
        p->rows.resize(n);
        p->nbytes.resize(n);
        p->dst_offset.resize(n);
    } catch (const std::bad_alloc&) {
        return fail(II_ENOMEM, "ii_plan: host allocation failed");
    }
    p->chunk_bytes = chunk_bytes;

    // 1. copy the table and compute byte sizes
    for (size_t i = 0; i < n; ++i) {
        const ii_tensor_desc& d = table[i];
        int w = width_of(d.dtype);
        if (!w) return fail(II_EINVAL, "ii_plan: row %zu: unknown dtype %d", i, d.dtype);
        if (d.ndim < 0 || (d.ndim > 0 && !d.shape))
            return fail(II_EINVAL, "ii_plan: row %zu: bad ndim/shape", i);
        if (!pow2(d.dst_align))
            return fail(II_EINVAL, "ii_plan: row %zu: dst_align %llu is not a power of two", i,
                        (unsigned long long)d.dst_align);
        uint64_t numel = 1;
        bool zero = false;
        p->shape_start[i] = p->shape_flat.size();
        for (int32_t k = 0; k < d.ndim; ++k) {
            if (d.shape[k] < 0) return fail(II_EINVAL, "ii_plan: row %zu: negative extent", i);
            p->shape_flat.push_back(d.shape[k]);
            uint64_t x = (uint64_t)d.shape[k];
            if (x == 0) zero = true;
        }
        if (zero) {
            numel = 0;
        } else {
            for (int32_t k = 0; k < d.ndim; ++k) {
                uint64_t x = (uint64_t)d.shape[k];
                if (__builtin_mul_overflow(numel, x, &numel))
                    return fail(II_EOVERFLOW, "ii_plan: row %zu: element count overflows", i);
            }
        }
        uint64_t nb;
        if (__builtin_mul_overflow(numel, (uint64_t)w, &nb))
            return fail(II_EOVERFLOW, "ii_plan: row %zu: byte size overflows", i);
        // rows: a strided tensor is shape[0] rows of rb bytes, row q at
        // src_offset + q * stride; every other non-empty tensor is one row
        uint64_t rows = nb ? 1 : 0, rb = nb;
        if (nb && d.src_row_stride) {
            if (d.ndim < 1)
                return fail(II_EINVAL, "ii_plan: row %zu: a row stride needs ndim >= 1", i);
            rows = (uint64_t)d.shape[0];
            rb = nb / rows;
            if (rows > 1 && d.src_row_stride < rb)
                return fail(II_EINVAL, "ii_plan: row %zu: row stride %llu is shorter than a row "
                            "(%llu bytes)", i, (unsigned long long)d.src_row_stride,
                            (unsigned long long)rb);
        }
        uint64_t last = d.src_offset, end;
        if (rows > 1) {
            uint64_t step;
            if (__builtin_mul_overflow(rows - 1, d.src_row_stride, &step) ||
                __builtin_add_overflow(d.src_offset, step, &last))
                return fail(II_EOVERFLOW, "ii_plan: row %zu: last row's offset overflows", i);
        }
        if (__builtin_add_overflow(last, rb, &end))
            return fail(II_EOVERFLOW, "ii_plan: row %zu: source end overflows", i);
        p->names[i] = d.name ? d.name : "";
        p->dtype[i] = d.dtype;
        p->ndim[i] = d.ndim;
        p->src_offset[i] = d.src_offset;
        p->dst_align[i] = d.dst_align;
        p->row_stride[i] = rows > 1 ? d.src_row_stride : 0;
        p->rows[i] = rows;
        p->nbytes[i] = nb;
        p->payload += nb;  // cannot overflow: disjoint ranges below 2^64
    }

    // 2. destination layout in table order
    {
        uint64_t end = 0, maxal = 1;
        for (size_t i = 0; i < n; ++i) {
            uint64_t a = p->dst_align[i], off;
            if (__builtin_add_overflow(end, a - 1, &off))
                return fail(II_EOVERFLOW, "ii_plan: destination layout overflows");
            off &= ~(a - 1);
            if (__builtin_add_overflow(off, p->nbytes[i], &end))
                return fail(II_EOVERFLOW, "ii_plan: destination layout overflows");
            p->dst_offset[i] = off;
            maxal = std::max(maxal, a);
        }
        uint64_t ar;
        if (__builtin_add_overflow(end, maxal - 1, &ar))
            return fail(II_EOVERFLOW, "ii_plan: arena size overflows");
        p->arena_bytes = ar & ~(maxal - 1);
        p->max_align = maxal;
    }

    // 3. source pieces in source order, overlap check, span
    std::vector<Piece> pieces;
    try {
        uint64_t total = 0;
        for (size_t i = 0; i < n; ++i) {
            total += p->rows[i];  // rows < 2^63, and the sum stops below 2^32
            if (total > (1ull << 31))
                return fail(II_EINVAL, "ii_plan: more than 2^31 rows in all");
        }
        pieces.reserve((size_t)total);
        for (size_t i = 0; i < n; ++i) {
            const uint64_t rows = p->rows[i];
            if (!rows) continue;
            const uint64_t rb = p->nbytes[i] / rows;
            for (uint64_t q = 0; q < rows; ++q)
                pieces.push_back(Piece{p->src_offset[i] + q * p->row_stride[i], rb, q * rb,
                                       (uint32_t)i});
        }
    } catch (const std::bad_alloc&) {
        return fail(II_ENOMEM, "ii_plan: host allocation failed");
    }
    // a table's own order is usually source order already
    if (!std::is_sorted(pieces.begin(), pieces.end(),
                        [](const Piece& a, const Piece& b) { return a.src < b.src; }))
        std::sort(pieces.begin(), pieces.end(),
                  [](const Piece& a, const Piece& b) { return a.src < b.src; });
    for (size_t j = 1; j < pieces.size(); ++j) {
        const Piece& a = pieces[j - 1];
        const Piece& b = pieces[j];
        if (b.src < a.src + a.len) {
            if (a.tensor == b.tensor)
                return fail(II_EOVERLAP, "ii_plan: rows of table row %u overlap", a.tensor);
            return fail(II_EOVERLAP, "ii_plan: source ranges of rows %u and %u overlap",
                        a.tensor, b.tensor);
        }
    }
    if (!pieces.empty()) {
        p->lo = pieces.front().src;
        p->hi = pieces.back().src + pieces.back().len;
    }
    const uint64_t C = chunk_bytes, lo = p->lo, span = p->hi - p->lo;
    p->num_chunks = span ? (size_t)((span - 1) / C + 1) : 0;
    if (p->num_chunks >= (1ull << 32))
        return fail(II_EINVAL, "ii_plan: more than 2^32 chunks");

    // 4. cut every piece at chunk boundaries, in source order
    try {
        size_t S = 0;
        for (const Piece& pc : pieces) {
            uint64_t b = pc.src - lo, e = b + pc.len;
            S += (size_t)((e - 1) / C - b / C + 1);
        }
        if (S >= (1ull << 32)) return fail(II_EINVAL, "ii_plan: more than 2^32 segments");
        p->seg_chunk.resize(S);
        p->seg_off.resize(S);
        p->seg_tensor.resize(S);
        p->seg_len.resize(S);
        p->seg_toff.resize(S);
        p->chunk_seg_begin.assign(p->num_chunks + 1, 0);
        size_t s = 0;
        for (const Piece& pc : pieces) {
            uint64_t b = pc.src - lo, e = b + pc.len;
            for (uint64_t x = b; x < e;) {
                uint64_t k = x / C, cend = std::min(e, (k + 1) * C);
                p->seg_chunk[s] = (uint32_t)k;
                p->seg_off[s] = (uint32_t)(x - k * C);
                p->seg_tensor[s] = pc.tensor;
                p->seg_len[s] = (uint32_t)(cend - x);
                p->seg_toff[s] = pc.toff + (x - b);
                p->chunk_seg_begin[k + 1]++;
                ++s;
                x = cend;
            }
        }
        std::vector<Piece>().swap(pieces);
        for (size_t k = 0; k < p->num_chunks; ++k)
            p->chunk_seg_begin[k + 1] += p->chunk_seg_begin[k];

        // 5. packed staging layout and gather runs
        p->seg_poff.resize(S);
        p->chunk_plen.assign(p->num_chunks, 0);
        p->chunk_run_begin.assign(p->num_chunks + 1, 0);
        for (size_t k = 0; k < p->num_chunks; ++k) {
            const uint64_t s0 = p->chunk_seg_begin[k], s1 = p->chunk_seg_begin[k + 1];
            uint64_t pos = 0;
            for (uint64_t x = s0; x < s1; ++x) {
                p->seg_poff[x] = (uint32_t)pos;
                if (p->seg_poff[x] != p->seg_off[x]) p->packed_distinct = true;
                const bool joins = x > s0 && p->seg_off[x - 1] + p->seg_len[x - 1] == p->seg_off[x];
                if (joins) {
                    p->run_len.back() += p->seg_len[x];
                } else {
                    p->run_off.push_back(p->seg_off[x]);
                    p->run_poff.push_back((uint32_t)pos);
                    p->run_len.push_back(p->seg_len[x]);
                }
                pos += p->seg_len[x];
            }
            p->chunk_plen[k] = pos;
            if (pos != p->chunk_len(k)) p->packed_distinct = true;
            p->chunk_run_begin[k + 1] = p->run_len.size();
        }
        // pinned blobs. A chunk whose runs form at most kMaxDmaGroups groups
        // of equal length and equal spacing (the rows of a column block,
        // whole tensor pieces) is moved by one copy per group straight into
        // the packed layout; otherwise it is gathered on the host when more
        // than a quarter of its used range is gaps, else its used range is
        // copied in place, gaps included. More copies per chunk would save
        // more host time but each adds a copy's start-up to the chunk
        // (measured on tensor-parallel shards: up to 2 groups beats both
        // the host gather and 8 groups).
        p->chunk_pinned.assign(p->num_chunks, kPinnedInPlace);
        if (p->packed_distinct) p->chunk_group_begin.assign(p->num_chunks + 1, 0);
        const uint32_t max_groups = env_u32("II_PINNED_GROUPS_MAX", kMaxDmaGroups, 0, 64);
        for (size_t k = 0; k < p->num_chunks; ++k) {
            uint64_t b, e;
            p->chunk_used(k, &b, &e);
            if (!p->packed_distinct) {
                p->copy_bytes += e - b;
                continue;
            }
            const uint64_t r0 = p->chunk_run_begin[k], r1 = p->chunk_run_begin[k + 1];
            const size_t g0 = p->groups.size();
            for (uint64_t r = r0; r < r1;) {
                DmaGroup g{p->run_off[r], p->run_poff[r], p->run_len[r], 1, 0};
                uint64_t q = r + 1;
                while (q < r1 && p->run_len[q] == g.len &&
                       (g.count == 1 || p->run_off[q] - p->run_off[q - 1] == g.stride)) {
                    g.stride = p->run_off[q] - p->run_off[q - 1];
                    ++g.count;
                    ++q;
                }
                p->groups.push_back(g);
                r = q;
            }
            uint8_t how = kPinnedInPlace;
            if (p->groups.size() - g0 <= max_groups) how = kPinnedGroups;
            else if (4 * (e - b - p->chunk_plen[k]) > (e - b)) how = kPinnedGather;
            if (how != kPinnedGroups) p->groups.resize(g0);
            p->chunk_group_begin[k + 1] = p->groups.size();
            p->chunk_pinned[k] = how;
            p->copy_bytes += how == kPinnedInPlace ? e - b : p->chunk_plen[k];
        }

        // 6. ring tiles: per chunk, tile_bytes of segment bytes each (packed
        // offsets), and -- for plans with gaps -- the same bytes as a window
        // of chunk offsets. Built segment by segment: the tiles that start
        // inside segment s begin their range at s, and every tile segment s
        // reaches has s in its range, so whole runs of tiles are filled at
        // once.
        uint32_t T = env_u32("II_TILE_BYTES", kDefaultTile, 1024, kMaxTile) & ~15u;
        p->tile_bytes = T;
        const std::vector<uint32_t>& po = p->seg_poff;
        p->chunk_tile_begin.assign(p->num_chunks + 1, 0);
        for (size_t k = 0; k < p->num_chunks; ++k)
            p->chunk_tile_begin[k + 1] = p->chunk_tile_begin[k] + (p->chunk_plen[k] + T - 1) / T;
        const uint64_t G = p->chunk_tile_begin[p->num_chunks];
        if (G > 0x7fffffffull) return fail(II_EINVAL, "ii_plan: more than 2^31 tiles");
        p->tiles.resize(G);
        if (p->packed_distinct) p->tile_win.resize(G);
        for (size_t k = 0; k < p->num_chunks; ++k) {
            const uint64_t s0 = p->chunk_seg_begin[k], s1 = p->chunk_seg_begin[k + 1];
            const uint64_t g0 = p->chunk_tile_begin[k];
            TileDev* td = p->tiles.data() + g0;
            for (uint64_t x = s0; x < s1; ++x) {
                const uint64_t P0 = po[x], P1 = P0 + p->seg_len[x];
                const uint64_t m0 = P0 / T, m1 = (P1 - 1) / T;
                // segment x is the first to meet tile m0 if it starts there
                if (P0 == m0 * T) td[m0].first = (uint32_t)x;
                td[m0].last = (uint32_t)(x + 1);
                if (m1 > m0) std::fill(td + m0 + 1, td + m1 + 1, TileDev{(uint32_t)x, (uint32_t)(x + 1)});
            }
            if (!p->packed_distinct) continue;
            // windows: tile m starts at the chunk offset of packed byte m*T,
            // which lies in segment first[m]; it ends where tile m+1 starts,
            // the chunk's last tile at its last segment's end
            const uint64_t M = p->chunk_tile_begin[k + 1] - g0;
            TileWin* tw = p->tile_win.data() + g0;
            for (uint64_t m = 0; m < M; ++m) {
                const uint32_t f = td[m].first;
                tw[m].w0 = (uint32_t)(p->seg_off[f] + (m * T - po[f]));
            }
            for (uint64_t m = 0; m + 1 < M; ++m) tw[m].w1 = tw[m + 1].w0;
            if (M) tw[M - 1].w1 = p->seg_off[s1 - 1] + p->seg_len[s1 - 1];
        }

        // 7. layout tiles: the segments in destination layout order, cut into
        // windows of T layout positions. Layout positions grow with the table
        // order and, inside a tensor, with the tensor offset, so a table read
        // in table order is already sorted. The windows a segment meets are
        // visited in increasing order; a window gets a tile the first time a
        // segment meets it, and later segments meeting it extend the tile's
        // range. Windows holding only padding get no tile.
        {
            std::vector<uint64_t> pos(S);
            for (size_t x = 0; x < S; ++x)
                pos[x] = p->dst_offset[p->seg_tensor[x]] + p->seg_toff[x];
            p->lseg.resize(S);
            for (size_t x = 0; x < S; ++x) p->lseg[x] = (uint32_t)x;
            auto by_pos = [&pos](uint32_t a, uint32_t b) { return pos[a] < pos[b]; };
            if (!std::is_sorted(pos.begin(), pos.end()))
                std::sort(p->lseg.begin(), p->lseg.end(), by_pos);
            uint64_t cur = ~0ull;  // window of the last tile made
            for (size_t j = 0; j < S; ++j) {
                const uint32_t x = p->lseg[j];
                const uint64_t m0 = pos[x] / T, m1 = (pos[x] + p->seg_len[x] - 1) / T;
                if (m1 >= (1ull << 32))
                    return fail(II_EINVAL, "ii_plan: destination layout beyond 2^32 tiles");
                for (uint64_t m = m0; m <= m1; ++m) {
                    if (m != cur) {
                        if (p->ltiles.size() >= 0x7fffffffull)
                            return fail(II_EINVAL, "ii_plan: more than 2^31 tiles");
                        p->ltiles.push_back(TileDev{(uint32_t)j, (uint32_t)(j + 1)});
                        p->lwin.push_back((uint32_t)m);
                        cur = m;
                    } else {
                        p->ltiles.back().last = (uint32_t)(j + 1);
                    }
                }
            }
            // windows strictly increase from window 0 or more: every window
            // holds segment bytes exactly when the last tile is window G - 1
            if (p->ltiles.empty() || p->lwin.back() == p->ltiles.size() - 1)
                std::vector<uint32_t>().swap(p->lwin);
            // The image kernel's variant for tables of many small tensors
            // (ii_plan_layout_mixed): when at least II_LAYOUT_MIXED_PCT
            // percent (default 5; 0 = always, 101 = never) of the tiles meet
            // three or more segments, or when at least 3% meet two or more
            // and most payload bytes are phase-shifted (their blob offset
            // and layout position differ mod 16, so each 16-byte block takes
            // two loads). The 100,000-tensor set has 10.4% tiles of three or
            // more; 20,000 byte-sized tensors of 16-256 KiB, 4.3% of two and
            // shifted bytes; a tensor-parallel shard of 4-15 KB rows, aligned
            // rows; tables of large tensors, none of either.
            uint64_t many = 0, two = 0, shifted = 0, bytes = 0;
            for (const TileDev& td : p->ltiles) {
                many += td.last - td.first >= 3;
                two += td.last - td.first >= 2;
            }
            for (size_t x = 0; x < S; ++x) {
                const uint64_t src = p->lo + (uint64_t)p->seg_chunk[x] * C + p->seg_off[x];
                bytes += p->seg_len[x];
                if ((src - pos[x]) & 15) shifted += p->seg_len[x];
            }
            const uint64_t G = p->ltiles.size();
            const uint32_t pct = env_u32("II_LAYOUT_MIXED_PCT", 5, 0, 101);
            p->layout_mixed = pct <= 100 && (many * 100 >= (uint64_t)pct * G ||
                                             (two * 100 >= 3 * G && shifted * 2 >= bytes));
        }
        p->na_rows.resize(S);
        p->na_ranges.reserve(n);
    } catch (const std::bad_alloc&) {
        return fail(II_ENOMEM, "ii_plan: host allocation failed");
    }

    p->ring_depth = env_u32("II_RING_DEPTH", 3, 1, 8);
    // lanes: as many as slots, up to 3 (with the caller's stream that is
    // the four hardware queues a process gets by default)
    p->copy_streams = std::min(p->ring_depth, env_u32("II_COPY_STREAMS", 3, 1, kMaxLanes));
    p->trace = env_u32("II_TRACE", 0, 0, 1) != 0;
    {
        long cores = sysconf(_SC_NPROCESSORS_ONLN);
        uint32_t dflt = (uint32_t)std::max(1L, std::min(8L, cores));
        p->host_threads = env_u32("II_HOST_THREADS", dflt, 1, 64);
    }
    *out = p.release();
    return II_OK;
}

extern "C" void ii_plan_free(ii_plan_t* plan) {
    if (!plan) return;
    runtime_destroy(plan);
    delete plan;
}

extern "C" size_t ii_plan_num_tensors(const ii_plan_t* p) { return p ? p->nbytes.size() : 0; }
extern "C" size_t ii_plan_num_chunks(const ii_plan_t* p) { return p ? p->num_chunks : 0; }
extern "C" size_t ii_plan_num_segments(const ii_plan_t* p) { return p ? p->seg_len.size() : 0; }
extern "C" uint64_t ii_plan_chunk_bytes(const ii_plan_t* p) { return p ? p->chunk_bytes : 0; }
extern "C" uint64_t ii_plan_payload_bytes(const ii_plan_t* p) { return p ? p->payload : 0; }
extern "C" uint64_t ii_plan_arena_bytes(const ii_plan_t* p) { return p ? p->arena_bytes : 0; }
extern "C" uint64_t ii_plan_copy_bytes(const ii_plan_t* p) { return p ? p->copy_bytes : 0; }

extern "C" void ii_plan_span(const ii_plan_t* p, uint64_t* lo, uint64_t* hi) {
    if (lo) *lo = p ? p->lo : 0;
    if (hi) *hi = p ? p->hi : 0;
}

extern "C" int ii_plan_tensors(const ii_plan_t* p, uint64_t* nbytes, uint64_t* dst_offset) {
    if (!p) return fail(II_EINVAL, "ii_plan_tensors: plan is NULL");
    size_t n = p->nbytes.size();
    if (nbytes && n) memcpy(nbytes, p->nbytes.data(), n * 8);
    if (dst_offset && n) memcpy(dst_offset, p->dst_offset.data(), n * 8);
    return II_OK;
}

extern "C" int ii_plan_chunks(const ii_plan_t* p, uint64_t* src_begin, uint64_t* len,
                              uint64_t* seg_begin) {
    if (!p) return fail(II_EINVAL, "ii_plan_chunks: plan is NULL");
    for (size_t k = 0; k < p->num_chunks; ++k) {
        if (src_begin) src_begin[k] = p->lo + k * p->chunk_bytes;
        if (len) len[k] = p->chunk_len(k);
    }
    if (seg_begin)
        for (size_t k = 0; k <= p->num_chunks; ++k) seg_begin[k] = p->chunk_seg_begin[k];
    return II_OK;
}

extern "C" int ii_plan_segments(const ii_plan_t* p, uint32_t* chunk, uint32_t* chunk_off,
                                uint32_t* tensor, uint64_t* tensor_off, uint32_t* len) {
    if (!p) return fail(II_EINVAL, "ii_plan_segments: plan is NULL");
    size_t S = p->seg_len.size();
    if (!S) return II_OK;
    if (chunk) memcpy(chunk, p->seg_chunk.data(), S * 4);
    if (chunk_off) memcpy(chunk_off, p->seg_off.data(), S * 4);
    if (tensor) memcpy(tensor, p->seg_tensor.data(), S * 4);
    if (tensor_off) memcpy(tensor_off, p->seg_toff.data(), S * 8);
    if (len) memcpy(len, p->seg_len.data(), S * 4);
    return II_OK;
}

extern "C" int ii_plan_tiles(const ii_plan_t* p, uint32_t* tile_bytes, uint64_t* num_tiles,
                             uint32_t* chunk, uint32_t* first, uint32_t* last, uint32_t* w0,
                             uint32_t* w1) {
    if (!p) return fail(II_EINVAL, "ii_plan_tiles: plan is NULL");
    if (tile_bytes) *tile_bytes = p->tile_bytes;
    if (num_tiles) *num_tiles = p->tiles.size();
    // gap-free plans keep no windows or chunk indices: tile m of chunk k is
    // the window [m * tile_bytes, ...) of the chunk
    for (size_t k = 0; k < p->num_chunks; ++k)
        for (uint64_t g = p->chunk_tile_begin[k]; g < p->chunk_tile_begin[k + 1]; ++g) {
            if (chunk) chunk[g] = (uint32_t)k;
            if (first) first[g] = p->tiles[g].first;
            if (last) last[g] = p->tiles[g].last;
            const uint64_t m = g - p->chunk_tile_begin[k];
            const uint64_t b = m * p->tile_bytes;
            if (w0) w0[g] = p->packed_distinct ? p->tile_win[g].w0 : (uint32_t)b;
            if (w1)
                w1[g] = p->packed_distinct ? p->tile_win[g].w1
                                           : (uint32_t)std::min<uint64_t>(p->chunk_len(k),
                                                                           b + p->tile_bytes);
        }
    return II_OK;
}

extern "C" int ii_plan_layout_tiles(const ii_plan_t* p, uint64_t* num_tiles, uint32_t* seg_order,
                                    uint32_t* first, uint32_t* last, uint32_t* window) {
    if (!p) return fail(II_EINVAL, "ii_plan_layout_tiles: plan is NULL");
    const size_t G = p->ltiles.size(), S = p->lseg.size();
    if (num_tiles) *num_tiles = G;
    if (seg_order && S) memcpy(seg_order, p->lseg.data(), S * 4);
    for (size_t g = 0; g < G; ++g) {
        if (first) first[g] = p->ltiles[g].first;
        if (last) last[g] = p->ltiles[g].last;
        if (window) window[g] = p->lwin.empty() ? (uint32_t)g : p->lwin[g];
    }
    return II_OK;
}

extern "C" int ii_plan_layout_mixed(const ii_plan_t* p) { return p && p->layout_mixed ? 1 : 0; }

extern "C" int ii_plan_packing(const ii_plan_t* p, uint32_t* seg_off, uint64_t* chunk_len) {
    if (!p) return fail(II_EINVAL, "ii_plan_packing: plan is NULL");
    const size_t S = p->seg_len.size();
    if (seg_off && S) memcpy(seg_off, p->seg_poff.data(), S * 4);
    if (chunk_len)
        for (size_t k = 0; k < p->num_chunks; ++k) chunk_len[k] = p->chunk_plen[k];
    return II_OK;
}

extern "C" const char* ii_plan_tensor_name(const ii_plan_t* p, size_t i) {
    if (!p || i >= p->names.size()) return "";
    return p->names[i].c_str();
}

extern "C" const char* ii_strerror(int status) {
    switch (status) {
    case II_OK: return "success";
    case II_EINVAL: return "invalid argument";
    case II_EOVERFLOW: return "size or offset overflows 64 bits";
    case II_EOVERLAP: return "overlapping ranges";
    case II_EALIGN: return "destination not aligned to dst_align";
    case II_ENOMEM: return "out of memory";
    case II_EARENA: return "arena too small";
    case II_EBUSY: return "plan in use by another call";
    case II_EHIP: return "HIP runtime error";
    case II_ERANGE: return "blob, image or file shorter than the plan's span";
    case II_EIO: return "reading the model file failed";
    case II_ESCRATCH: return "plan tables exceed the static workspace";
    default: return "unknown status";
    }
}

extern "C" const char* ii_last_error(void) { return g_last_error.c_str(); }
