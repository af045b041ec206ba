// Which memory the device may touch: the decision behind the destination
// and image checks of every load, kept apart from the HIP queries that feed
// it so that it can be exercised on the host.
#pragma once

#include <cstddef>
#include <cstdint>
#include <vector>

#include "ii_internal.h"

namespace ii {

// What the runtime reports about the allocation that holds an address.
struct AllocInfo {
    enum Kind { kUnknown = 0, kDevice = 1, kPinnedHost = 2 } kind = kUnknown;
    bool extent = false;  // whether [base, base + size) is known
    uint64_t base = 0, size = 0;
};

// Whether the device may touch [b, e), given what is reported for address
// b: the whole range must lie inside that one allocation. Pageable host
// memory and unknown addresses are never reachable; a pinned host range
// whose allocation extent is not reported is refused; device memory whose
// extent is not reported is accepted (it is device memory at b, and nothing
// better is known).
inline bool reachable(const AllocInfo& a, uint64_t b, uint64_t e) {
    if (a.kind == AllocInfo::kUnknown) return false;
    if (!a.extent) return a.kind == AllocInfo::kDevice;
    return b >= a.base && e <= a.base + a.size;
}

// The first range of v (sorted by address) that the device may not touch,
// or v.size(). info(addr) reports the allocation holding addr; a range that
// lies inside the allocation found last needs no further query, so ranges
// packed into one arena cost one query.
template <class Info>
size_t first_unreachable(const std::vector<DstRange>& v, Info&& info) {
    uint64_t ab = 0, ae = 0;  // extent of the allocation found last
    for (size_t j = 0; j < v.size(); ++j) {
        const DstRange& d = v[j];
        if (d.b >= ab && d.e <= ae) continue;
        const AllocInfo a = info(d.b);
        if (!reachable(a, d.b, d.e)) return j;
        if (a.extent) {
            ab = a.base;
            ae = a.base + a.size;
        } else {
            ab = ae = 0;
        }
    }
    return v.size();
}

}  // namespace ii
