// The host copy pool under ThreadSanitizer: many copies of varied sizes
// (below and above the split threshold), several pool sizes, every byte
// checked, and pools created and destroyed repeatedly.
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

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
    printf("OK\n");
    return 0;
}
