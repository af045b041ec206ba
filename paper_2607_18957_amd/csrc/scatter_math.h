// Per-lane arithmetic of the scatter kernel, written once for the device
// kernel and for the host-side emulator that checks it (every address it
// forms is bounds-checked on the CPU before the kernel ever runs).
//
// Terms (see scatter.hip for the full description):
//   row    one segment staged for a tile: where its bytes go and come from;
//   unit   one (segment, 16-byte-aligned destination block) pair;
//   anchor the source offset of the first destination byte a unit covers; a
//          unit belongs to the tile whose window holds its anchor.
#pragma once

#include <cstdint>

#if defined(__HIPCC__)
#define II_HD __host__ __device__ inline __attribute__((always_inline))
#else
#define II_HD inline
#endif

namespace ii {

constexpr uint32_t kBlock = 128;           // threads per scatter workgroup
constexpr int kUnroll = 2;                 // units in flight per lane
constexpr uint32_t kMaxSegBatch = kBlock;  // segment rows staged in LDS at once
constexpr uint32_t kMaxTile = 64u << 10;   // largest tile a workgroup takes
// Largest workgroup count of one launch: a dispatch counts its grid in
// work-items, in 32 bits.
constexpr uint32_t kMaxGridBlocks = 0xffffffffu / kBlock;

// One dispatch over n workgroups (n < 2^32): a dispatch counts each grid
// dimension in 32-bit work-items, so the grid is gy rows of gx workgroups,
// gx * kBlock <= 2^32 - 1, and workgroup (x, y) takes index y * gx + x;
// indices from n up to gx * gy - 1 (fewer than gy of them) have no work.
II_HD void grid_shape(uint64_t n, uint32_t* gx, uint32_t* gy) {
    const uint64_t y = n ? (n + kMaxGridBlocks - 1) / kMaxGridBlocks : 1;
    *gy = (uint32_t)y;
    *gx = (uint32_t)(n ? (n + y - 1) / y : 1);
}

struct SegRow {
    uint64_t delta;  // source address minus destination address
    uint64_t dbeg;   // destination range [dbeg, dend)
    uint64_t dend;
    uint64_t ubase;  // destination block index of the row's unit 0, minus its prefix
};

// A segment whose first byte sits at chunk offset off, whose len bytes go to
// destination address dst, seen from the tile window [w0, w1) of a chunk that
// starts at source address cbase: the row and the number of its units the
// tile owns.
II_HD SegRow make_row(uint64_t dst, uint64_t off, uint64_t len, uint64_t cbase, uint64_t w0,
                      uint64_t w1, uint32_t* count) {
    const uint64_t b0 = dst >> 4;
    const uint64_t nunits = ((dst + len + 15) >> 4) - b0;
    // units whose anchor lies before chunk offset x
    uint64_t u0 = 0, u1 = 0;
    if (w0 > off) {
        const uint64_t c = ((dst + (w0 - off) + 15) >> 4) - b0;
        u0 = c < nunits ? c : nunits;
    }
    if (w1 > off) {
        const uint64_t c = ((dst + (w1 - off) + 15) >> 4) - b0;
        u1 = c < nunits ? c : nunits;
    }
    *count = (uint32_t)(u1 - u0);
    SegRow r;
    r.delta = cbase + off - dst;
    r.dbeg = dst;
    r.dend = dst + len;
    r.ubase = b0 + u0;
    return r;
}

// Index of the row that owns tile unit u: the last row whose exclusive
// prefix is <= u (rows with no units share their successor's prefix and are
// skipped by this rule). pre[0] == 0 and u < total.
II_HD uint32_t find_row(const uint32_t* pre, uint32_t nrows, uint32_t u) {
    uint32_t lo = 0, hi = nrows;
    while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) >> 1;
        if (pre[mid] <= u) lo = mid;
        else hi = mid;
    }
    return lo;
}

// Everything a lane needs to move one unit: destination block address d; the
// covered bytes [c0, c1) of that block; the aligned source words to load
// (word0 at A, word1 at A + 16, each only if it holds a needed byte); and the
// byte phase p of the block's source inside word0.
struct UnitIO {
    uint64_t d;
    uint64_t A;
    uint32_t c0, c1;
    uint32_t p;
    bool need0, need1;
};

II_HD UnitIO unit_io(const SegRow& r, uint64_t unit_in_tile) {
    UnitIO io;
    io.d = (r.ubase + unit_in_tile) << 4;
    const uint64_t ds = io.d > r.dbeg ? io.d : r.dbeg;
    const uint64_t de = (io.d + 16) < r.dend ? io.d + 16 : r.dend;
    const uint64_t a = io.d + r.delta;  // source address of destination byte d
    io.A = a & ~15ull;
    io.p = (uint32_t)(a & 15u);
    io.c0 = (uint32_t)(ds - io.d);
    io.c1 = (uint32_t)(de - io.d);
    io.need0 = ds + r.delta < io.A + 16;  // first needed source byte is in word0
    io.need1 = de + r.delta > io.A + 16;  // last needed source byte is in word1
    return io;
}

struct U4 {
    uint32_t x, y, z, w;
};

II_HD uint32_t funnel32(uint32_t hi, uint32_t lo, uint32_t bytes) {
    return (uint32_t)((((uint64_t)hi << 32) | lo) >> (8u * bytes));
}

// Bytes p .. p+15 (p in 0..15) of the 32-byte little-endian value hi:lo.
II_HD U4 funnel16(U4 lo, U4 hi, uint32_t p) {
    const uint32_t q = p >> 2, r = p & 3u;
    const bool q0 = q == 0, q1 = q == 1, q2 = q == 2;
    const uint32_t e0 = q0 ? lo.x : q1 ? lo.y : q2 ? lo.z : lo.w;
    const uint32_t e1 = q0 ? lo.y : q1 ? lo.z : q2 ? lo.w : hi.x;
    const uint32_t e2 = q0 ? lo.z : q1 ? lo.w : q2 ? hi.x : hi.y;
    const uint32_t e3 = q0 ? lo.w : q1 ? hi.x : q2 ? hi.y : hi.z;
    const uint32_t e4 = q0 ? hi.x : q1 ? hi.y : q2 ? hi.z : hi.w;
    U4 o;
    o.x = funnel32(e1, e0, r);
    o.y = funnel32(e2, e1, r);
    o.z = funnel32(e3, e2, r);
    o.w = funnel32(e4, e3, r);
    return o;
}

II_HD uint32_t dword_at(U4 v, uint32_t i) {
    return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w;
}

// Store bytes [c0, c1) of block v at block address d (d 16-aligned) with the
// widest naturally aligned stores inside [c0, c1). Mem provides st16, st8,
// st4, st2, st1 taking an address and a value.
template <class Mem>
II_HD void store_unit(Mem& m, uint64_t d, U4 v, uint32_t c0, uint32_t c1) {
    if (c0 == 0 && c1 == 16) {
        m.st16(d, v);
        return;
    }
    while (c0 < c1) {
        const uint32_t room = c1 - c0;
        if ((c0 & 7u) == 0 && room >= 8) {
            const uint32_t i = c0 >> 2;
            m.st8(d + c0, dword_at(v, i), dword_at(v, i + 1));
            c0 += 8;
        } else if ((c0 & 3u) == 0 && room >= 4) {
            m.st4(d + c0, dword_at(v, c0 >> 2));
            c0 += 4;
        } else if ((c0 & 1u) == 0 && room >= 2) {
            m.st2(d + c0, (uint16_t)(dword_at(v, c0 >> 2) >> (8u * (c0 & 3u))));
            c0 += 2;
        } else {
            m.st1(d + c0, (uint8_t)(dword_at(v, c0 >> 2) >> (8u * (c0 & 3u))));
            c0 += 1;
        }
    }
}

}  // namespace ii
