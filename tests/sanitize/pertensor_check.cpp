// The per-tensor path's host schedule (pertensor.h) on the host: every
// staging copy, every host-to-device copy and every slot hand-over it asks
// for is checked against the buffers it names; the staging copies are
// carried out on host memory and every device copy is checked to move
// exactly the bytes of its tensor that the blob holds at those offsets. Built with AddressSanitizer and
// UndefinedBehaviorSanitizer; prints OK or the first failed check.
//
// Cases: the 100,000-tensor stress table (sizes log-uniform in [64 B, 64 KiB),
// widths 1/2/4, sources in a permuted order, 16 MiB slots, ring depth 3 --
// the table of the per-tensor runs), small slots that every tensor
// straddles, tensors given as rows at a stride, and random tables.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <numeric>
#include <random>
#include <vector>

#include "pertensor.h"

namespace {

struct Table {
    std::vector<uint64_t> nbytes, rows, stride, src;  // stride 0: contiguous
    uint64_t blob_bytes = 0;
};

int failures = 0;
char first_failure[512];

void fail(const char* what, uint64_t a, uint64_t b) {
    if (!failures++)
        snprintf(first_failure, sizeof first_failure, "%s (%llu, %llu)", what,
                 (unsigned long long)a, (unsigned long long)b);
}

// Run the schedule over host buffers and check it. A device copy is carried
// out as a comparison: the slot bytes it would move must be the tensor's own
// bytes at those offsets, read from the blob by the tensor's definition (row
// q, byte c at src + q * stride + c); pieces must arrive in tensor order, each
// tensor front to back without gap or overlap, so at the end every byte of
// every tensor has been moved exactly once.
void check(const Table& t, uint64_t slot_bytes, uint32_t depth, uint64_t* copies_out) {
    const size_t n = t.nbytes.size();
    // blob bytes: a function of the position
    std::vector<uint8_t> blob(t.blob_bytes);
    for (uint64_t x = 0; x < blob.size(); ++x) blob[x] = (uint8_t)(x * 2654435761u >> 13);
    std::vector<std::vector<uint8_t>> slots(depth, std::vector<uint8_t>(slot_bytes));
    std::vector<uint64_t> moved(n, 0);  // bytes of each tensor moved so far
    // the slot being filled; bytes of it staged since it was taken
    uint32_t open = 0;
    std::vector<uint8_t> staged(slot_bytes, 0);
    uint64_t copies = 0, last_tensor = 0, last_end = 0;
    bool any = false;

    auto stage = [&](uint32_t slot, uint64_t at, size_t i, uint64_t src_rel, uint64_t len) -> int {
        if (slot != open) fail("stage into a slot that is not open", slot, open);
        if (i >= n) fail("stage for a tensor out of range", i, n);
        if (!len || at + len > slot_bytes) fail("stage outside the slot", at, len);
        // the source bytes must lie inside one row of tensor i
        const uint64_t rb = t.nbytes[i] / t.rows[i];
        const uint64_t q = t.stride[i] ? src_rel / t.stride[i] : 0;
        const uint64_t c = t.stride[i] ? src_rel % t.stride[i] : src_rel;
        if (q >= t.rows[i] || c + len > rb) fail("stage source outside the tensor's rows", i, src_rel);
        if (t.src[i] + src_rel + len > blob.size()) fail("stage source outside the blob", i, src_rel);
        if (failures) return 1;
        memcpy(slots[slot].data() + at, blob.data() + t.src[i] + src_rel, len);
        for (uint64_t x = at; x < at + len; ++x) {
            if (staged[x]) fail("slot byte staged twice in one fill", slot, x);
            staged[x] = 1;
        }
        return failures ? 1 : 0;
    };
    auto copy = [&](uint32_t slot, uint64_t at, size_t i, uint64_t toff, uint64_t len) -> int {
        if (slot != open) fail("copy from a slot that is not open", slot, open);
        if (i >= n || !len || toff + len > t.nbytes[i]) fail("copy outside the tensor", i, toff);
        if (at + len > slot_bytes) fail("copy outside the slot", at, len);
        if (failures) return 1;
        for (uint64_t x = at; x < at + len; ++x)
            if (!staged[x]) fail("copy of a slot byte not staged in this fill", slot, x);
        // pieces come in tensor order, each tensor front to back
        if (any && (i < last_tensor || (i == last_tensor && toff != last_end)))
            fail("pieces out of order", i, toff);
        if (i != last_tensor && toff != 0) fail("tensor does not start at byte 0", i, toff);
        any = true;
        last_tensor = i;
        last_end = toff + len;
        if (toff != moved[i]) fail("piece does not continue its tensor", i, toff);
        const uint64_t rb = t.nbytes[i] / t.rows[i];
        for (uint64_t x = 0; x < len && !failures; ++x) {
            const uint64_t y = toff + x, q = y / rb, c = y % rb;
            if (slots[slot][at + x] != blob[t.src[i] + q * t.stride[i] + c])
                fail("a device copy would move bytes that are not the tensor's", i, y);
        }
        moved[i] = toff + len;
        ++copies;
        return failures ? 1 : 0;
    };
    auto close = [&](uint32_t slot, uint32_t next) -> int {
        if (slot != open) fail("close of a slot that is not open", slot, open);
        if (next != depth && next != (slot + 1) % depth) fail("slots not taken round robin", slot, next);
        if (next < depth) {
            open = next;  // the caller waits for its last copies before refilling it
            std::fill(staged.begin(), staged.end(), 0);
        } else {
            open = depth;
        }
        return failures ? 1 : 0;
    };
    const int rc = ii::pertensor_schedule(t.nbytes.data(), t.rows.data(), t.stride.data(), n,
                                          slot_bytes, depth, stage, copy, close);
    if (rc && !failures) fail("schedule returned an error", rc, 0);
    if (failures) return;
    for (size_t i = 0; i < n; ++i)
        if (moved[i] != t.nbytes[i]) {
            fail("tensor not moved whole", i, moved[i]);
            return;
        }
    if (open != depth && copies) fail("the last slot was not closed", open, depth);
    if (copies_out) *copies_out = copies;
}

Table stress_like(uint64_t n, uint32_t seed) {
    std::mt19937_64 g(seed);
    std::uniform_real_distribution<double> u(std::log(64.0), std::log(65536.0));
    const uint64_t widths[3] = {4, 2, 1};
    Table t;
    for (uint64_t i = 0; i < n; ++i) {
        const uint64_t b = (uint64_t)std::floor(std::exp(u(g))), w = widths[g() % 3];
        t.nbytes.push_back(std::max<uint64_t>(1, b / w) * w);
        t.rows.push_back(1);
        t.stride.push_back(0);
    }
    std::vector<uint64_t> perm(n);
    std::iota(perm.begin(), perm.end(), 0);
    std::shuffle(perm.begin(), perm.end(), g);
    t.src.assign(n, 0);
    uint64_t at = 0;
    for (uint64_t i : perm) {
        t.src[i] = at;
        at += t.nbytes[i];
    }
    t.blob_bytes = at;
    return t;
}

Table random_table(std::mt19937_64& g) {
    Table t;
    const uint64_t n = 1 + g() % 40;
    uint64_t at = g() % 100;
    for (uint64_t i = 0; i < n; ++i) {
        const uint64_t kind = g() % 4;
        if (kind == 0) {  // empty
            t.nbytes.push_back(0);
            t.rows.push_back(0);
            t.stride.push_back(0);
            t.src.push_back(at);
        } else if (kind == 1) {  // rows at a stride
            const uint64_t rows = 1 + g() % 9, rb = 1 + g() % 300, stride = rb + g() % 200;
            t.nbytes.push_back(rows * rb);
            t.rows.push_back(rows);
            t.stride.push_back(rows > 1 ? stride : 0);
            t.src.push_back(at);
            at += (rows - 1) * stride + rb + g() % 50;
        } else {
            const uint64_t nb = 1 + g() % 5000;
            t.nbytes.push_back(nb);
            t.rows.push_back(1);
            t.stride.push_back(0);
            t.src.push_back(at);
            at += nb + g() % 50;
        }
    }
    t.blob_bytes = at + 1;
    return t;
}

}  // namespace

int main() {
    uint64_t copies = 0;
    // the stress-shaped table of the per-tensor runs: 16 MiB slots, depth 3
    const Table s = stress_like(100000, 2);
    check(s, 16u << 20, 3, &copies);
    if (!failures && copies < 100000) fail("fewer copies than tensors", copies, 100000);
    // slots smaller than most tensors (every tensor straddles slots), depth 1 and 2
    const Table small = stress_like(3000, 5);
    check(small, 4096, 1, nullptr);
    check(small, 4096 + 16, 2, nullptr);
    check(small, 64, 8, nullptr);
    // random tables: empty tensors, rows at a stride, gaps, slot sizes 1 .. 9000
    std::mt19937_64 g(2026);
    for (int it = 0; it < 3000 && !failures; ++it) {
        const Table t = random_table(g);
        check(t, 1 + g() % 9000, 1 + (uint32_t)(g() % 8), nullptr);
    }
    if (failures) {
        printf("FAIL: %s (%d failures)\n", first_failure, failures);
        return 1;
    }
    printf("OK copies=%llu\n", (unsigned long long)copies);
    return 0;
}
