// The reachability decision of the loads (reach.h) against a fake memory
// map: device and pinned host allocations, with and without a reported
// extent, side by side and with pageable holes between them. Built with
// AddressSanitizer and UndefinedBehaviorSanitizer; prints OK or the first
// failed case.
#include <cstdio>
#include <vector>

#include "reach.h"

using ii::AllocInfo;
using ii::DstRange;

namespace {

struct Fake {
    struct A {
        uint64_t b, e;
        AllocInfo::Kind kind;
        bool extent;
    };
    std::vector<A> allocs;
    mutable int queries = 0;
    AllocInfo operator()(uint64_t x) const {
        ++queries;
        AllocInfo i;
        for (const A& a : allocs)
            if (x >= a.b && x < a.e) {
                i.kind = a.kind;
                i.extent = a.extent;
                if (a.extent) {
                    i.base = a.b;
                    i.size = a.e - a.b;
                }
            }
        return i;
    }
};

int failures = 0;

void expect(bool cond, const char* what) {
    if (!cond) {
        printf("FAIL: %s\n", what);
        ++failures;
    }
}

size_t run(const Fake& f, std::vector<DstRange> v) {
    f.queries = 0;
    return ii::first_unreachable(v, std::cref(f));
}

}  // namespace

int main() {
    const uint64_t K = 1 << 16;
    Fake f;
    f.allocs = {
        {0x100000, 0x100000 + K, AllocInfo::kDevice, true},
        {0x200000, 0x200000 + K, AllocInfo::kPinnedHost, true},
        {0x200000 + K, 0x200000 + 2 * K, AllocInfo::kPinnedHost, true},  // right after
        {0x300000, 0x300000 + K, AllocInfo::kPinnedHost, true},          // after a hole
        {0x400000, 0x400000 + K, AllocInfo::kPinnedHost, false},         // extent unknown
        {0x500000, 0x500000 + K, AllocInfo::kDevice, false},             // extent unknown
        {0x600000, 0x600000 + K, AllocInfo::kDevice, true},
    };
    // one range per case
    struct Case {
        uint64_t b, e;
        bool ok;
        const char* what;
    } cases[] = {
        {0x100000, 0x100000 + K, true, "whole device allocation"},
        {0x100010, 0x100020, true, "inside a device allocation"},
        {0x100000, 0x100000 + K + 1, false, "one byte past a device allocation"},
        {0x200000, 0x200000 + K, true, "whole pinned allocation"},
        {0x200000 + K - 8, 0x200000 + K + 8, false, "across two adjacent pinned allocations"},
        {0x200000, 0x300000 + K, false, "from a pinned allocation over a hole into another"},
        {0x200000 + 2 * K, 0x200000 + 2 * K + 16, false, "pageable memory"},
        {0x400000, 0x400010, false, "pinned allocation with unknown extent"},
        {0x500000, 0x500010, true, "device allocation with unknown extent"},
        {0x50, 0x60, false, "unknown address"},
        {0x600000 + K - 1, 0x600000 + K, true, "last byte of an allocation"},
    };
    for (const Case& c : cases) {
        const size_t j = run(f, {{c.b, c.e, 0}});
        expect((j == 1) == c.ok, c.what);
    }
    // many ranges in one allocation: one query; the first bad one is named
    std::vector<DstRange> v;
    for (uint64_t x = 0; x < 64; ++x) v.push_back({0x100000 + x * 256, 0x100000 + x * 256 + 200, x});
    expect(run(f, v) == v.size() && f.queries == 1, "ranges in one allocation, one query");
    v.push_back({0x200000, 0x200100, 64});
    v.push_back({0x200100, 0x200200, 65});
    expect(run(f, v) == v.size() && f.queries == 2, "two allocations, two queries");
    v.push_back({0x200000 + K - 4, 0x200000 + K + 4, 66});
    expect(run(f, v) == 66, "a later range crossing into the next allocation is found");
    // after an allocation with unknown extent nothing is taken as known
    std::vector<DstRange> w = {{0x500000, 0x500010, 0}, {0x500020, 0x500030, 1},
                               {0x600000, 0x600010, 2}};
    expect(run(f, w) == w.size() && f.queries == 3, "unknown extent is queried per range");
    if (failures) return 1;
    printf("OK\n");
    return 0;
}
