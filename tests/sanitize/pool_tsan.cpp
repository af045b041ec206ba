// The host copy pool under ThreadSanitizer: many copies of varied sizes
// (below and above the split threshold), several pool sizes, every byte
// checked, and pools created and destroyed repeatedly; file reads,
// read-ahead, and gathers of many runs from memory and from a file.
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <unistd.h>
#include <vector>
#include <algorithm>

#include "copy_pool.h"

int main() {
    std::vector<uint8_t> src(20u << 20), dst(20u << 20);
    for (size_t i = 0; i < src.size(); ++i) src[i] = (uint8_t)(i * 2654435761u >> 13);
    const uint64_t sizes[] = {0, 1, 4095, 4u << 20, (4u << 20) + 17, 13u << 20, 20u << 20};
    for (uint32_t threads : {1u, 2u, 3u, 8u}) {
        ii::CopyPool pool(threads);
        for (int rep = 0; rep < 3; ++rep)
            for (uint64_t n : sizes) {
                const uint64_t off = (uint64_t)rep * 7 % 64;
                if (n + off > src.size()) continue;
                std::fill(dst.begin(), dst.end(), 0xEE);
                pool.copy(dst.data(), src.data() + off, n);
                if (n && memcmp(dst.data(), src.data() + off, n) != 0) {
                    fprintf(stderr, "mismatch (n=%llu threads=%u)\n", (unsigned long long)n,
                            threads);
                    return 2;
                }
                if (n < dst.size() && dst[n] != 0xEE) {
                    fprintf(stderr, "write past the end (n=%llu)\n", (unsigned long long)n);
                    return 2;
                }
            }
    }
    // file reads: whole, unaligned, past the end of the file (allowed beyond
    // `need`), and an early end (EIO)
    char path[] = "/tmp/ii_pool_tsanXXXXXX";
    const int fd = mkstemp(path);
    if (fd < 0) return 3;
    const uint64_t fsz = (9u << 20) + 123;
    if (write(fd, src.data(), fsz) != (ssize_t)fsz) return 3;
    for (uint32_t threads : {1u, 3u, 8u}) {
        ii::CopyPool pool(threads);
        struct Case { uint64_t off, len, need; int want; } cases[] = {
            {0, fsz, fsz, 0}, {4096, 8u << 20, 8u << 20, 0}, {17, (5u << 20) + 5, (5u << 20) + 5, 0},
            {8u << 20, 2u << 20, fsz - (8u << 20), 0}, {8u << 20, 2u << 20, 2u << 20, EIO}};
        for (const Case& c : cases) {
            std::fill(dst.begin(), dst.end(), 0xEE);
            const int err = pool.read(fd, dst.data(), c.off, c.len, 4096, c.need);
            if (err != c.want) {
                fprintf(stderr, "read(%llu, %llu): err %d, want %d\n", (unsigned long long)c.off,
                        (unsigned long long)c.len, err, c.want);
                return 2;
            }
            const uint64_t have = std::min(c.len, fsz - c.off);
            if (!err && memcmp(dst.data(), src.data() + c.off, have) != 0) {
                fprintf(stderr, "read mismatch off=%llu\n", (unsigned long long)c.off);
                return 2;
            }
        }
    }
    // read-ahead: all chunks in order (several thread counts), stopping
    // halfway, and a file that ends early
    const uint64_t C = 1u << 20;
    const uint32_t K = (uint32_t)((fsz + C - 1) / C);
    auto range = [&](uint32_t k) {
        const uint64_t at = (uint64_t)k * C, len = std::min(C, fsz - at);
        return ii::ReadAhead::Range{at, at + len, len};
    };
    for (uint32_t threads : {1u, 2u, 5u, 8u}) {
        for (int stop_early = 0; stop_early < 2; ++stop_early) {
            ii::ReadAhead ra(fd, threads, C, K, range);
            if (!ra.ok()) return 3;
            for (uint32_t k = 0; k < K; ++k) {
                if (stop_early && k == K / 2) break;
                int err = 0;
                const uint8_t* b = ra.wait(k, &err);
                const uint64_t len = std::min(C, fsz - (uint64_t)k * C);
                if (!b || err || memcmp(b, src.data() + (uint64_t)k * C, len) != 0) {
                    fprintf(stderr, "read-ahead chunk %u wrong (threads %u)\n", k, threads);
                    return 2;
                }
                ra.release(k);
            }
        }
    }
    {
        auto past = [&](uint32_t k) {  // asks for one chunk more than the file has
            const uint64_t at = (uint64_t)k * C;
            return ii::ReadAhead::Range{at, at + C, C};
        };
        ii::ReadAhead ra(fd, 3, C, K + 1, past);
        int err = 0;
        for (uint32_t k = 0; k <= K; ++k) {
            const uint8_t* b = ra.wait(k, &err);
            if (!b) break;
            ra.release(k);
        }
        if (err != EIO) {
            fprintf(stderr, "read-ahead past the end: err %d, want EIO\n", err);
            return 2;
        }
    }
    // gathers: many runs (rows of a sharded tensor) from memory and from the
    // file, split across threads by destination bytes; every byte checked
    // against a one-run-at-a-time copy, nothing written past the end. Run
    // patterns: rows of up to 9000 bytes with short gaps; thousands of tiny
    // runs (a file batch fills its iovecs and starts another); and groups of
    // runs separated by gaps longer than a file batch reads through
    struct Pattern { uint64_t span; uint32_t gap_mod, run_mod, big_gap_every; };
    const Pattern patterns[] = {{6u << 20, 700, 9000, 0}, {96u << 10, 32, 16, 0},
                                {8u << 20, 700, 9000, 200}};
    for (const Pattern& pat : patterns) {
        std::vector<uint32_t> off, poff, len;
        uint64_t s = 0, total = 0;
        uint32_t x = 12345;
        while (s < pat.span) {
            x = x * 1103515245u + 12345u;
            uint32_t gap = (x >> 8) % pat.gap_mod;
            const uint32_t run = 1 + (x >> 16) % pat.run_mod;
            if (pat.big_gap_every && off.size() % pat.big_gap_every == pat.big_gap_every - 1)
                gap += 300u << 10;
            s += gap;
            off.push_back((uint32_t)s);
            poff.push_back((uint32_t)total);
            len.push_back(run);
            s += run;
            total += run;
        }
        if (4096 + s > fsz || total >= dst.size()) return 3;  // inside the file and dst
        const int64_t skews[] = {0, (int64_t)off[0], -64};  // b0[0] at, past, before offset 0
        for (uint32_t threads : {1u, 3u, 8u}) {
            ii::CopyPool pool(threads);
            for (int64_t skew : skews) {
                std::vector<uint8_t> want(total);
                // b0[0] holds source offset `skew`: source offset o is b0[o - skew]
                const uint8_t* b0 = src.data() + 4096;
                for (size_t r = 0; r < off.size(); ++r)
                    memcpy(want.data() + poff[r], b0 + ((int64_t)off[r] - skew), len[r]);
                std::fill(dst.begin(), dst.end(), 0xEE);
                pool.gather(dst.data(), b0, skew, off.data(), poff.data(), len.data(), off.size(),
                            total);
                if (memcmp(dst.data(), want.data(), total) != 0 || dst[total] != 0xEE) {
                    fprintf(stderr, "gather mismatch (threads %u skew %lld)\n", threads,
                            (long long)skew);
                    return 2;
                }
                if (skew) continue;
                std::fill(dst.begin(), dst.end(), 0xEE);
                const int err = pool.read_gather(fd, dst.data(), 4096, off.data(), poff.data(),
                                                 len.data(), off.size(), total);
                if (err || memcmp(dst.data(), want.data(), total) != 0 || dst[total] != 0xEE) {
                    fprintf(stderr, "read_gather mismatch (threads %u err %d)\n", threads, err);
                    return 2;
                }
                // a base past the end of the file: EIO
                if (pool.read_gather(fd, dst.data(), fsz, off.data(), poff.data(), len.data(),
                                     off.size(), total) != EIO) {
                    fprintf(stderr, "read_gather past the end did not fail\n");
                    return 2;
                }
            }
        }
    }
    close(fd);
    unlink(path);
    printf("OK\n");
    return 0;
}
