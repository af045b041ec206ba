// The host-side schedule of the naive per-tensor pipeline (Sec. 4.2, "Naive
// CFA Model"), kept apart from the HIP calls that carry it out so that every
// range it forms can be checked on the host.
//
// Tensors go in table order. Each tensor's bytes (its rows back to back, for
// a tensor given as rows) are cut into pieces that fit the rest of the
// current staging slot; a piece is staged (host copies of whole row parts
// from the blob into the slot) and then moved by one host-to-device copy
// into the tensor's destination. A slot is filled piece after piece until
// it is full; then it is closed and the next slot (round robin over
// `depth`) is taken, once the copies that last read it have finished.
#pragma once

#include <algorithm>
#include <cstddef>
#include <cstdint>

namespace ii {

// Callbacks, each returning 0 or an error code that ends the schedule:
//   stage(slot, slot_off, i, src_rel, len)  copy len blob bytes starting src_rel
//                                           bytes past tensor i's source offset
//                                           into slot + slot_off
//   copy(slot, slot_off, i, toff, len)      one DMA: slot + slot_off -> dst[i] + toff
//   close(slot, next)                       slot is full (or the last): its
//                                           copies are recorded; next is the
//                                           slot to be filled after it, to be
//                                           waited for if it was used before
//                                           (next == depth: no slot follows)
template <class Stage, class Copy, class Close>
int pertensor_schedule(const uint64_t* nbytes, const uint64_t* rows, const uint64_t* row_stride,
                       size_t n, uint64_t slot_bytes, uint32_t depth, Stage&& stage, Copy&& copy,
                       Close&& close) {
    uint32_t slot = 0;
    uint64_t used = 0;  // bytes of the current slot already packed
    for (size_t i = 0; i < n; ++i) {
        const uint64_t nb = nbytes[i];
        if (!nb) continue;
        const uint64_t rb = nb / rows[i], stride = row_stride[i];
        for (uint64_t x = 0; x < nb;) {
            if (used == slot_bytes) {
                const uint32_t next = (slot + 1) % depth;
                if (int rc = close(slot, next)) return rc;
                slot = next;
                used = 0;
            }
            // tensor bytes [x, x + len): row q from byte c, row by row
            const uint64_t len = std::min(nb - x, slot_bytes - used);
            for (uint64_t y = x; y < x + len;) {
                const uint64_t q = y / rb, c = y % rb, m = std::min(x + len - y, rb - c);
                if (int rc = stage(slot, used + (y - x), i, q * stride + c, m)) return rc;
                y += m;
            }
            if (int rc = copy(slot, used, i, x, len)) return rc;
            used += len;
            x += len;
        }
    }
    if (used) return close(slot, depth);
    return 0;
}

}  // namespace ii
