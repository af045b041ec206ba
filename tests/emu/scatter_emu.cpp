// CPU emulation of the scatter kernel, with every memory access checked.
//
// Test infrastructure. It drives the kernel's own per-lane arithmetic
// (scatter_math.h: rows, unit ownership, lane -> row search, aligned-word
// loads, byte funnel, exact edge stores) through the same tile / batch / unit
// loop as scatter_chunks, one lane after another, against emulated memory:
//   * a load is legal only if its 16-byte word holds at least one source byte
//     of the row being copied (the kernel's no-fault guarantee);
//   * a store is legal only inside the row's destination range;
//   * every destination byte of every tensor must be written exactly once.
// Violations are reported as text; results go into a host arena the tests
// compare with the oracle.
#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "scatter_math.h"

using namespace ii;

namespace {

constexpr uint32_t kBlockE = kBlock;  // the kernel's workgroup size
constexpr int kUnrollE = kUnroll;     // the kernel's units per lane

struct EmuMem {
    // source: chunk bytes, addressed as src_base + (k * C) + off
    const uint8_t* blob = nullptr;
    uint64_t lo = 0, hi = 0;
    uint64_t src_base = 0;  // emulated address of span byte lo
    // destination arena
    uint8_t* arena = nullptr;
    uint64_t arena_base = 0, arena_len = 0;
    std::vector<uint8_t>* writes = nullptr;
    // the row currently being copied
    uint64_t row_src_b = 0, row_src_e = 0, row_dst_b = 0, row_dst_e = 0;
    std::string err;
    uint64_t loads = 0, stores = 0;

    void bad(const char* what, uint64_t a) {
        if (err.empty()) {
            char b[256];
            snprintf(b, sizeof b, "%s at %#llx (row src [%#llx,%#llx) dst [%#llx,%#llx))", what,
                     (unsigned long long)a, (unsigned long long)row_src_b,
                     (unsigned long long)row_src_e, (unsigned long long)row_dst_b,
                     (unsigned long long)row_dst_e);
            err = b;
        }
    }
    uint8_t src_byte(uint64_t a) {
        // bytes of the same 16-byte word outside the span read as 0xEE
        uint64_t x = a - src_base + lo;
        if (a < src_base || x >= hi) return 0xEE;
        return blob[x];
    }
    U4 ld16(uint64_t a) {
        ++loads;
        if (a & 15) bad("unaligned 16-byte load", a);
        if (!(a < row_src_e && row_src_b < a + 16)) bad("load of a word with no source byte", a);
        uint8_t b[16];
        for (int i = 0; i < 16; ++i) b[i] = src_byte(a + i);
        U4 v;
        memcpy(&v, b, 16);
        return v;
    }
    void put(uint64_t a, const uint8_t* b, int n, int align) {
        ++stores;
        if (a % align) bad("misaligned store", a);
        for (int i = 0; i < n; ++i) {
            uint64_t x = a + i;
            if (x < row_dst_b || x >= row_dst_e) {
                bad("store outside the row's destination", x);
                continue;
            }
            if (x < arena_base || x - arena_base >= arena_len) {
                bad("store outside the arena", x);
                continue;
            }
            arena[x - arena_base] = b[i];
            (*writes)[x - arena_base]++;
        }
    }
    void st16(uint64_t a, U4 v) { put(a, reinterpret_cast<const uint8_t*>(&v), 16, 16); }
    void st8(uint64_t a, uint32_t lo_, uint32_t hi_) {
        uint32_t w[2] = {lo_, hi_};
        put(a, reinterpret_cast<const uint8_t*>(w), 8, 8);
    }
    void st4(uint64_t a, uint32_t v) { put(a, reinterpret_cast<const uint8_t*>(&v), 4, 4); }
    void st2(uint64_t a, uint16_t v) { put(a, reinterpret_cast<const uint8_t*>(&v), 2, 2); }
    void st1(uint64_t a, uint8_t v) { put(a, &v, 1, 1); }
};

}  // namespace

extern "C" {

// Emulate every tile, in the plan's tile order. Segment rows and tiles are
// the plan's (as exported by the C-ABI); dst_addr are emulated destination
// addresses inside [arena_base, arena_base + arena_len); src_base is the
// emulated address of span byte lo (chunk k starts at src_base + k*C).
// packed = 0: each tile's window [w0, w1) of chunk offsets applies, as in a
// resident image; packed = 1: seg_off are packed slot offsets and tile m of
// chunk k takes [m * tile_bytes, ...) up to chunk_plen[k], as in a packed
// staging slot; per_chunk != 0 (resident image of a gap-free table): as the
// kernel does, tile g is window g % per_chunk of chunk g / per_chunk and
// tile_chunk / w0 / w1 are not read. Returns 0 if every check held, else 1
// with a message in err.
int emu_scatter(uint64_t num_chunks, uint64_t chunk_bytes, uint64_t lo, uint64_t hi,
                const uint8_t* blob, const uint32_t* seg_off, const uint32_t* seg_len,
                const uint32_t* seg_tensor, const uint64_t* seg_toff, uint64_t ntiles,
                const uint32_t* tile_chunk, const uint32_t* tile_first, const uint32_t* tile_last,
                const uint32_t* tile_w0, const uint32_t* tile_w1, int packed, uint32_t per_chunk,
                uint32_t tile_bytes,
                const uint64_t* chunk_plen, const uint64_t* tensor_dst,
                const uint64_t* tensor_nbytes, uint64_t ntensors, uint64_t src_base,
                uint64_t arena_base, uint64_t arena_len, uint8_t* arena, uint32_t batch, char* err,
                int errlen, uint64_t* stats) {
    EmuMem m;
    m.blob = blob;
    m.lo = lo;
    m.hi = hi;
    m.src_base = src_base;
    m.arena = arena;
    m.arena_base = arena_base;
    m.arena_len = arena_len;
    std::vector<uint8_t> writes(arena_len, 0);
    m.writes = &writes;
    uint64_t units = 0, max_rows = 0;
    std::vector<SegRow> rows(batch);
    if (batch > kMaxSegBatch) batch = kMaxSegBatch;
    std::vector<uint32_t> pre(batch), cnt(batch), srow(batch);

    uint64_t tile_in_chunk = 0;
    for (uint64_t g = 0; g < ntiles && m.err.empty(); ++g) {
        uint64_t k, w0, w1;
        if (per_chunk) {
            k = g / per_chunk;
            const uint64_t clen =
                (k + 1 == num_chunks) ? (hi - lo) - chunk_bytes * k : chunk_bytes;
            w0 = (g - k * per_chunk) * (uint64_t)tile_bytes;
            w1 = std::min<uint64_t>(clen, w0 + tile_bytes);
        } else {
            k = tile_chunk[g];
            w0 = tile_w0[g];
            w1 = tile_w1[g];
        }
        if (k >= num_chunks) {
            m.bad("tile of a chunk out of range", k);
            break;
        }
        tile_in_chunk = (g && tile_chunk[g - 1] == k) ? tile_in_chunk + 1 : 0;
        const uint64_t cbase = src_base + k * chunk_bytes;
        if (packed) {
            w0 = tile_in_chunk * tile_bytes;
            w1 = std::min<uint64_t>(chunk_plen[k], w0 + tile_bytes);
        }
        {
            const uint32_t first = tile_first[g], last = tile_last[g];
            max_rows = std::max<uint64_t>(max_rows, last - first);
            for (uint32_t s0 = first; s0 < last && m.err.empty(); s0 += batch) {
                const uint32_t ns = std::min(batch, last - s0);
                uint32_t total = 0;
                for (uint32_t i = 0; i < ns; ++i) {
                    const uint32_t s = s0 + i;
                    const uint64_t dst = tensor_dst[seg_tensor[s]] + seg_toff[s];
                    rows[i] = make_row(dst, seg_off[s], seg_len[s], cbase, w0, w1, &cnt[i]);
                    pre[i] = total;
                    total += cnt[i];
                    rows[i].ubase -= pre[i];
                    srow[i] = s;
                }
                // lanes exactly as the kernel runs them: kBlock lanes, each with
                // kUnroll units at stride kBlock, rows found in lock step
                for (uint32_t base = 0; base < total && m.err.empty(); base += kBlockE * kUnrollE) {
                    for (uint32_t tid = 0; tid < kBlockE && m.err.empty(); ++tid) {
                        for (int j = 0; j < kUnrollE; ++j) {
                            const uint32_t u = base + (uint32_t)j * kBlockE + tid;
                            if (u >= total || !m.err.empty()) continue;
                            const uint32_t r = find_row(pre.data(), ns, u);
                            if (r >= ns) m.bad("row index out of range", r);
                            if (!(pre[r] <= u && u < pre[r] + cnt[r])) {
                                m.bad("lane mapped to a row that does not own its unit", u);
                                break;
                            }
                            const uint32_t s = srow[r];
                            m.row_src_b = cbase + seg_off[s];
                            m.row_src_e = m.row_src_b + seg_len[s];
                            m.row_dst_b = rows[r].dbeg;
                            m.row_dst_e = rows[r].dend;
                            const UnitIO io = unit_io(rows[r], u);
                            // the unit's anchor must lie in this tile
                            const uint64_t first_src = io.d + io.c0 + rows[r].delta - cbase;
                            if (first_src < w0 || first_src >= w1)
                                m.bad("unit anchored outside its tile", io.d);
                            U4 x0{0, 0, 0, 0}, x1{0, 0, 0, 0};
                            if (io.need0) x0 = m.ld16(io.A);
                            if (io.need1) x1 = m.ld16(io.A + 16);
                            const U4 v = funnel16(x0, x1, io.p);
                            if (io.c1 > io.c0) store_unit(m, io.d, v, io.c0, io.c1);
                            else m.bad("unit with no bytes", io.d);
                            ++units;
                        }
                    }
                }
            }
        }
    }
    // every tensor byte exactly once, nothing else
    if (m.err.empty()) {
        std::vector<uint8_t> want(arena_len, 0);
        for (uint64_t i = 0; i < ntensors; ++i) {
            if (!tensor_nbytes[i]) continue;
            uint64_t b = tensor_dst[i] - arena_base;
            for (uint64_t j = 0; j < tensor_nbytes[i]; ++j) want[b + j] = 1;
        }
        for (uint64_t x = 0; x < arena_len; ++x)
            if (writes[x] != want[x]) {
                char b[160];
                snprintf(b, sizeof b, "arena byte %llu written %u times, expected %u",
                         (unsigned long long)x, writes[x], want[x]);
                m.err = b;
                break;
            }
    }
    if (stats) {
        stats[0] = units;
        stats[1] = m.loads;
        stats[2] = m.stores;
        stats[3] = max_rows;
    }
    if (!m.err.empty()) {
        snprintf(err, errlen, "%s", m.err.c_str());
        return 1;
    }
    return 0;
}

// Emulate the resident-image kernel (scatter_layout) over the plan's layout
// tiles. (Its single-segment path forms the one row in every lane and maps
// lane unit u to unit u of that row: the arithmetic below with one row,
// whose prefix is 0, so this emulation covers both paths.) Tile g takes the layout positions [window[g] * tile_bytes, +
// tile_bytes) and the layout-order segments seg_order[first[g] ..
// last[g]); segment x's bytes sit at emulated address src_base + chunk[x] *
// chunk_bytes + chunk_off[x] and go to tensor_dst[tensor[x]] + tensor_off[x],
// its layout position being dst_offset[tensor[x]] + tensor_off[x]. Checks
// as emu_scatter, and that every unit's anchor (the layout position of its
// first destination byte) lies in its tile's window.
int emu_scatter_layout(uint64_t chunk_bytes, uint64_t lo, uint64_t hi, const uint8_t* blob,
                       const uint32_t* seg_chunk, const uint32_t* seg_off,
                       const uint32_t* seg_len, const uint32_t* seg_tensor,
                       const uint64_t* seg_toff, const uint32_t* seg_order, uint64_t ntiles,
                       const uint32_t* tile_first, const uint32_t* tile_last,
                       const uint32_t* tile_window, uint32_t tile_bytes,
                       const uint64_t* tensor_dst, const uint64_t* tensor_dst_offset,
                       const uint64_t* tensor_nbytes, uint64_t ntensors, uint64_t src_base,
                       uint64_t arena_base, uint64_t arena_len, uint8_t* arena, uint32_t batch,
                       char* err, int errlen, uint64_t* stats) {
    EmuMem m;
    m.blob = blob;
    m.lo = lo;
    m.hi = hi;
    m.src_base = src_base;
    m.arena = arena;
    m.arena_base = arena_base;
    m.arena_len = arena_len;
    std::vector<uint8_t> writes(arena_len, 0);
    m.writes = &writes;
    uint64_t units = 0, max_rows = 0;
    if (batch > kMaxSegBatch) batch = kMaxSegBatch;
    std::vector<SegRow> rows(batch);
    std::vector<uint32_t> pre(batch), cnt(batch), srow(batch);
    std::vector<uint64_t> rpos(batch), rdst(batch);
    uint64_t prev_window = 0;
    for (uint64_t g = 0; g < ntiles && m.err.empty(); ++g) {
        const uint64_t w0 = (uint64_t)tile_window[g] * tile_bytes, w1 = w0 + tile_bytes;
        if (g && tile_window[g] <= prev_window) m.bad("tile windows not increasing", g);
        prev_window = tile_window[g];
        const uint32_t first = tile_first[g], last = tile_last[g];
        if (first >= last) m.bad("tile without segments", g);
        max_rows = std::max<uint64_t>(max_rows, last - first);
        for (uint32_t s0 = first; s0 < last && m.err.empty(); s0 += batch) {
            const uint32_t ns = std::min(batch, last - s0);
            uint32_t total = 0;
            for (uint32_t i = 0; i < ns; ++i) {
                const uint32_t s = seg_order[s0 + i];
                const uint64_t src = (uint64_t)seg_chunk[s] * chunk_bytes + seg_off[s];
                rdst[i] = tensor_dst[seg_tensor[s]] + seg_toff[s];
                rpos[i] = tensor_dst_offset[seg_tensor[s]] + seg_toff[s];
                rows[i] = make_row(rdst[i], rpos[i], seg_len[s], src_base + src - rpos[i], w0,
                                   w1, &cnt[i]);
                pre[i] = total;
                total += cnt[i];
                rows[i].ubase -= pre[i];
                srow[i] = s;
            }
            for (uint32_t base = 0; base < total && m.err.empty(); base += kBlockE * kUnrollE) {
                for (uint32_t tid = 0; tid < kBlockE && m.err.empty(); ++tid) {
                    for (int j = 0; j < kUnrollE; ++j) {
                        const uint32_t u = base + (uint32_t)j * kBlockE + tid;
                        if (u >= total || !m.err.empty()) continue;
                        const uint32_t r = find_row(pre.data(), ns, u);
                        if (r >= ns) m.bad("row index out of range", r);
                        if (!(pre[r] <= u && u < pre[r] + cnt[r])) {
                            m.bad("lane mapped to a row that does not own its unit", u);
                            break;
                        }
                        const uint32_t s = srow[r];
                        m.row_src_b = src_base + (uint64_t)seg_chunk[s] * chunk_bytes + seg_off[s];
                        m.row_src_e = m.row_src_b + seg_len[s];
                        m.row_dst_b = rows[r].dbeg;
                        m.row_dst_e = rows[r].dend;
                        const UnitIO io = unit_io(rows[r], u);
                        const uint64_t anchor = rpos[r] + (io.d + io.c0 - rdst[r]);
                        if (anchor < w0 || anchor >= w1) m.bad("unit anchored outside its tile", io.d);
                        U4 x0{0, 0, 0, 0}, x1{0, 0, 0, 0};
                        if (io.need0) x0 = m.ld16(io.A);
                        if (io.need1) x1 = m.ld16(io.A + 16);
                        const U4 v = funnel16(x0, x1, io.p);
                        if (io.c1 > io.c0) store_unit(m, io.d, v, io.c0, io.c1);
                        else m.bad("unit with no bytes", io.d);
                        ++units;
                    }
                }
            }
        }
    }
    if (m.err.empty()) {
        std::vector<uint8_t> want(arena_len, 0);
        for (uint64_t i = 0; i < ntensors; ++i) {
            if (!tensor_nbytes[i]) continue;
            uint64_t b = tensor_dst[i] - arena_base;
            for (uint64_t j = 0; j < tensor_nbytes[i]; ++j) want[b + j] = 1;
        }
        for (uint64_t x = 0; x < arena_len; ++x)
            if (writes[x] != want[x]) {
                char b[160];
                snprintf(b, sizeof b, "arena byte %llu written %u times, expected %u",
                         (unsigned long long)x, writes[x], want[x]);
                m.err = b;
                break;
            }
    }
    if (stats) {
        stats[0] = units;
        stats[1] = m.loads;
        stats[2] = m.stores;
        stats[3] = max_rows;
    }
    if (!m.err.empty()) {
        snprintf(err, errlen, "%s", m.err.c_str());
        return 1;
    }
    return 0;
}

// The image launch's grid for n workgroups (grid_shape): no dimension may
// count more than 2^32 - 1 work-items, the indices y * gx + x must cover
// [0, n), and fewer than gy of them may lie past it. Returns 0 if so.
int emu_grid_check(uint64_t n, uint32_t* gx_out, uint32_t* gy_out) {
    uint32_t gx, gy;
    grid_shape(n, &gx, &gy);
    *gx_out = gx;
    *gy_out = gy;
    const uint64_t cover = (uint64_t)gx * gy;
    if ((uint64_t)gx * kBlock > 0xffffffffull || (uint64_t)gy * 1 > 0xffffffffull) return 1;
    if (cover < n || (n && cover - n >= gy) || gx == 0 || gy == 0) return 1;
    if (cover - 1 > 0xffffffffull) return 1;  // the kernel forms indices in 32 bits
    return 0;
}

}  // extern "C"
