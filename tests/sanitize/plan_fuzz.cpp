// Planner under AddressSanitizer + UndefinedBehaviorSanitizer (host only).
//
// Builds random tables -- including zero-size tensors, scalars, huge
// extents that overflow, overlapping and touching ranges, every dtype and
// alignment, tensors given as strided rows and column blocks whose rows
// interleave -- plans them with several chunk sizes, reads every getter and
// checks the structural invariants that need no oracle: segments tile each
// tensor exactly, lie inside their chunk and inside one row, and are
// ordered; tiles take tile_bytes of segment bytes each with contiguous
// windows; the copied bytes lie between the payload and the span; a pinned
// chunk's group copies rebuild the packed layout of its runs. Any sanitizer
// report or failed check exits non-zero.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <vector>

#include "ii.h"
#include "ii_internal.h"

namespace ii {
void runtime_destroy(ii_plan_t*) {}  // no device state in a host-only build
}

static uint64_t rng_state = 88172645463325252ull;
static uint64_t rnd() {  // xorshift64
    rng_state ^= rng_state << 13;
    rng_state ^= rng_state >> 7;
    rng_state ^= rng_state << 17;
    return rng_state;
}
static uint64_t pick(uint64_t n) { return rnd() % n; }

#define CHECK(c)                                                         \
    do {                                                                 \
        if (!(c)) {                                                      \
            fprintf(stderr, "check failed: %s (line %d)\n", #c, __LINE__); \
            exit(2);                                                     \
        }                                                                \
    } while (0)

int main(int argc, char** argv) {
    const int iters = argc > 1 ? atoi(argv[1]) : 3000;
    int ok_plans = 0, errors = 0;
    for (int it = 0; it < iters; ++it) {
        const size_t n = pick(40);
        std::vector<std::vector<int64_t>> shapes(n);
        std::vector<ii_tensor_desc> t(n, ii_tensor_desc{});
        static const uint64_t width[11] = {0, 1, 1, 1, 1, 2, 2, 4, 4, 8, 8};
        uint64_t pos = pick(64);
        if (pick(3) == 0) {
            // column blocks of one [R, row] byte matrix: rows of all tensors interleave
            const uint64_t R = 1 + pick(6);
            uint64_t col = 0;
            std::vector<uint64_t> w(n);
            for (size_t i = 0; i < n; ++i) w[i] = 1 + pick(9);
            uint64_t row = pick(4);
            for (size_t i = 0; i < n; ++i) row += w[i];
            for (size_t i = 0; i < n; ++i) {
                shapes[i] = {(int64_t)R, (int64_t)w[i]};
                t[i].name = nullptr;
                t[i].dtype = 1;
                t[i].ndim = 2;
                t[i].shape = shapes[i].data();
                t[i].dst_align = 1ull << pick(9);
                t[i].src_offset = pos + col;
                t[i].src_row_stride = row;
                col += w[i];
            }
        } else {
            for (size_t i = 0; i < n; ++i) {
                const int nd = (int)pick(4);
                for (int d = 0; d < nd; ++d) shapes[i].push_back(pick(10) ? (int64_t)pick(50) : 0);
                t[i].name = (i % 3) ? "w" : nullptr;
                t[i].dtype = 1 + (int32_t)pick(10);
                t[i].ndim = (int32_t)shapes[i].size();
                t[i].shape = shapes[i].empty() ? nullptr : shapes[i].data();
                t[i].dst_align = 1ull << pick(13);
                t[i].src_offset = pos;
                t[i].src_row_stride = 0;
                uint64_t numel = 1;
                for (int64_t x : shapes[i]) numel *= (uint64_t)x;
                const uint64_t nb = numel * width[t[i].dtype];
                if (nd >= 1 && nb && pick(3) == 0) {  // strided rows with gaps
                    const uint64_t rows = (uint64_t)shapes[i][0], rb = nb / rows;
                    t[i].src_row_stride = rb + pick(20);
                    pos += (rows - 1) * t[i].src_row_stride + rb;
                } else {
                    pos += nb;
                }
                pos += pick(3) ? 0 : pick(40);
            }
        }
        // one table in four gets one bad row of a random kind
        if (n && pick(4) == 0) {
            const size_t i = pick(n);
            switch (pick(10)) {
            case 0: t[i].dtype = pick(2) ? 0 : 11; break;                   // unknown dtype
            case 1: shapes[i].push_back(-1); break;                           // negative extent
            case 2: shapes[i].push_back((int64_t)(1ull << 40));               // size overflows
                    shapes[i].push_back((int64_t)(1ull << 40)); break;
            case 3: t[i].dst_align = 3; break;                                // not a power of two
            case 4: t[i].src_offset = ~0ull - pick(100); break;               // end overflows
            case 5: if (i) t[i].src_offset = t[i - 1].src_offset; break;      // overlap (if non-empty)
            case 6: t[i].ndim = -1; break;
            case 7: t[i].src_row_stride = 1; break;                           // rows overlap (if > 1 row of > 1 byte)
            case 8: t[i].src_row_stride = ~0ull / 2; break;                   // last row overflows (if > 2 rows)
            case 9: shapes[i].clear(); t[i].src_row_stride = 8; break;        // strided scalar
            }
            t[i].shape = shapes[i].empty() ? nullptr : shapes[i].data();
            if (t[i].ndim >= 0) t[i].ndim = (int32_t)shapes[i].size();
        }
        const uint64_t chunks[] = {16, 32, 48, 64, 4096, 1 << 16, 0, 17};
        for (uint64_t C : chunks) {
            ii_plan_t* p = nullptr;
            int rc = ii_plan(t.data(), n, C, &p);
            if (rc) {
                CHECK(p == nullptr);
                CHECK(ii_last_error()[0] != 0);
                ++errors;
                continue;
            }
            ++ok_plans;
            const size_t N = ii_plan_num_tensors(p), K = ii_plan_num_chunks(p),
                         S = ii_plan_num_segments(p);
            CHECK(N == n);
            std::vector<uint64_t> nb(N), off(N), cb(K), cl(K), sb(K + 1);
            std::vector<uint32_t> sc(S), so(S), st(S), sl(S);
            std::vector<uint64_t> sto(S);
            CHECK(ii_plan_tensors(p, nb.data(), off.data()) == 0);
            CHECK(ii_plan_chunks(p, cb.data(), cl.data(), sb.data()) == 0);
            CHECK(ii_plan_segments(p, sc.data(), so.data(), st.data(), sto.data(), sl.data()) == 0);
            uint32_t tb = 0;
            uint64_t G = 0;
            CHECK(ii_plan_tiles(p, &tb, &G, nullptr, nullptr, nullptr, nullptr, nullptr) == 0);
            std::vector<uint32_t> tk(G), tf(G), tl(G), tw0(G), tw1(G);
            CHECK(ii_plan_tiles(p, &tb, &G, tk.data(), tf.data(), tl.data(), tw0.data(),
                                tw1.data()) == 0);
            std::vector<uint32_t> spo(S);
            std::vector<uint64_t> plen(K);
            CHECK(ii_plan_packing(p, spo.data(), plen.data()) == 0);
            for (size_t i = 0; i < N; ++i) (void)ii_plan_tensor_name(p, i);
            uint64_t lo, hi;
            ii_plan_span(p, &lo, &hi);
            // rows of each tensor as the table gives them
            std::vector<uint64_t> rows(N), rb(N);
            for (size_t i = 0; i < N; ++i) {
                rows[i] = nb[i] ? (t[i].src_row_stride ? (uint64_t)shapes[i][0] : 1) : 0;
                rb[i] = rows[i] ? nb[i] / rows[i] : 0;
            }
            // segments: inside their chunk and one row, ordered, and tiling each tensor
            std::vector<uint64_t> covered(N, 0);
            uint64_t total = 0;
            for (size_t s = 0; s < S; ++s) {
                CHECK(sc[s] < K && st[s] < N && sl[s] > 0);
                CHECK((uint64_t)so[s] + sl[s] <= cl[sc[s]]);
                const uint64_t q = sto[s] / rb[st[s]], c = sto[s] % rb[st[s]];
                CHECK(c + sl[s] <= rb[st[s]]);
                CHECK(cb[sc[s]] + so[s] ==
                      t[st[s]].src_offset + q * (rows[st[s]] > 1 ? t[st[s]].src_row_stride : 0) + c);
                CHECK(sto[s] == covered[st[s]]);  // source order = offset order within a tensor
                covered[st[s]] += sl[s];
                total += sl[s];
                if (s && sc[s] == sc[s - 1]) CHECK(so[s] >= so[s - 1] + sl[s - 1]);
                if (s) CHECK(sc[s] >= sc[s - 1]);
            }
            for (size_t i = 0; i < N; ++i) CHECK(covered[i] == nb[i]);
            CHECK(total == ii_plan_payload_bytes(p));
            CHECK(ii_plan_copy_bytes(p) >= total && ii_plan_copy_bytes(p) <= hi - lo);
            for (size_t k = 0; k < K; ++k) CHECK(sb[k] <= sb[k + 1]);
            // tiles: in chunk order; per chunk ceil(plen / tb) of them; windows
            // contiguous from the first segment to the last segment's end;
            // segment windows inside the chunk's segments and advancing
            size_t g = 0;
            for (size_t k = 0; k < K; ++k) {
                uint64_t plen_k = 0;
                for (uint64_t s = sb[k]; s < sb[k + 1]; ++s) {
                    CHECK(spo[s] == plen_k);
                    plen_k += sl[s];
                }
                CHECK(plen[k] == plen_k);
                const uint64_t M = (plen_k + tb - 1) / tb;
                for (uint64_t m = 0; m < M; ++m, ++g) {
                    CHECK(g < G && tk[g] == k);
                    CHECK(sb[k] <= tf[g] && tf[g] < tl[g] && tl[g] <= sb[k + 1]);
                    CHECK(tw0[g] < tw1[g] && tw1[g] <= cl[k]);
                    if (m == 0) CHECK(tw0[g] == so[sb[k]]);
                    else CHECK(tw0[g] == tw1[g - 1] && tf[g] >= tf[g - 1]);
                    if (m + 1 == M) CHECK(tw1[g] == so[sb[k + 1] - 1] + sl[sb[k + 1] - 1]);
                }
            }
            CHECK(g == G);
            // pinned-blob moves: a grouped chunk's copies (rows of len bytes
            // every stride bytes, landing back to back) rebuild exactly the
            // packed layout the host gather makes from the chunk's runs;
            // copy_bytes sums what each chunk's move carries
            {
                const ii_plan_s* ip = p;
                uint64_t moved = 0;
                for (size_t k = 0; k < K; ++k) {
                    uint64_t ub, ue;
                    ip->chunk_used(k, &ub, &ue);
                    if (!ip->packed_distinct) {
                        moved += ue - ub;
                        continue;
                    }
                    const uint8_t how = ip->chunk_pinned[k];
                    const uint64_t g0 = ip->chunk_group_begin[k], g1 = ip->chunk_group_begin[k + 1];
                    const uint64_t r0 = ip->chunk_run_begin[k], r1 = ip->chunk_run_begin[k + 1];
                    moved += how == ii::kPinnedInPlace ? ue - ub : plen[k];
                    if (how != ii::kPinnedGroups) {
                        CHECK(g0 == g1);
                        if (how == ii::kPinnedGather) CHECK(4 * (ue - ub - plen[k]) > ue - ub);
                        continue;
                    }
                    const char* gm = getenv("II_PINNED_GROUPS_MAX");
                    CHECK(g1 - g0 <= (gm && *gm ? strtoull(gm, nullptr, 10) : ii::kMaxDmaGroups));
                    std::vector<uint8_t> chunk(cl[k]), a(plen[k], 0xEE), b(plen[k], 0xDD);
                    for (uint64_t x = 0; x < cl[k]; ++x) chunk[x] = (uint8_t)(x * 131 + k * 7 + 1);
                    for (uint64_t r = r0; r < r1; ++r) {
                        CHECK((uint64_t)ip->run_off[r] + ip->run_len[r] <= cl[k]);
                        CHECK((uint64_t)ip->run_poff[r] + ip->run_len[r] <= plen[k]);
                        for (uint32_t y = 0; y < ip->run_len[r]; ++y)
                            a[ip->run_poff[r] + y] = chunk[ip->run_off[r] + y];
                    }
                    uint64_t rows = 0;
                    for (uint64_t gi = g0; gi < g1; ++gi) {
                        const ii::DmaGroup& gr = ip->groups[gi];
                        CHECK(gr.count >= 1 && gr.len > 0);
                        if (gr.count > 1) CHECK(gr.stride > gr.len);
                        CHECK((uint64_t)gr.off + (uint64_t)(gr.count - 1) * gr.stride + gr.len <= cl[k]);
                        CHECK((uint64_t)gr.poff + (uint64_t)gr.count * gr.len <= plen[k]);
                        for (uint32_t q = 0; q < gr.count; ++q)
                            for (uint32_t y = 0; y < gr.len; ++y)
                                b[gr.poff + (uint64_t)q * gr.len + y] =
                                    chunk[gr.off + (uint64_t)q * gr.stride + y];
                        rows += gr.count;
                    }
                    CHECK(rows == r1 - r0);
                    CHECK(a == b);
                }
                CHECK(moved == ii_plan_copy_bytes(p));
            }
            ii_plan_free(p);
        }
    }
    printf("OK plans=%d rejected=%d\n", ok_plans, errors);
    return 0;
}
