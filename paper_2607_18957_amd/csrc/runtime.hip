// Load pipeline: pinned staging ring, bulk host-to-device copies and
// per-chunk scatters on the ring's lanes (its own streams), hipEvent edges
// between them, and the C-ABI entry points that drive it.
//
// The chunk lifecycle of InstantInfer's refined tensor materialisation
// (arXiv 2607.18957, Sec. 4.2) maps onto the ring as follows; j counts the
// chunks that hold at least one segment (the others are never touched), and
// chunk j's copy and scatter both run on lane j mod L.
//   InDisk -> InMem   host threads bring chunk j's bytes into pinned slot
//                     j mod D: a copy of its used range, or a gather of only
//                     its segments when it has gaps (pageable blob or file;
//                     a pinned blob is copied by DMA straight from itself,
//                     row group by row group when a chunk with gaps has few
//                     of them, and gathered on the host only when it has
//                     many and is mostly gaps). The slot is reused only once
//                     the copy that last read it has finished: host wait on
//                     copy_done[slot].
//   InMem  -> InGPU   one hipMemcpyAsync per chunk (or one per row group,
//                     2-D for rows at a fixed stride) into device slot
//                     j mod D on the chunk's lane; with one lane the copies
//                     run back to back in chunk order (the paper's
//                     (C_i,InGPU)->(C_i+1,InMem) edge). The device slot is
//                     free once the scatter that last read it is done: the
//                     lane's own stream order, or scatter_done[slot] when
//                     another lane ran that scatter. Records copy_done[slot].
//   InGPU  -> tensors the scatter kernel over the chunk's tiles, next on the
//                     same lane, moving its tensor pieces from Alloc to
//                     Loaded; records scatter_done[slot].
//   Destroyed         scatter_done[slot] releases the slot to chunk j + D.
// The caller's stream gates the first write into destination memory: lane
// 0 waits for an entry event recorded on it before its first scatter (and
// runs a switch's scrub), the other lanes wait for lane 0's `go` event; the
// copies into the ring need no such wait. At the end lane 0 joins the other
// lanes and the caller's stream waits for its done event, so the load is
// ordered on that stream like any other stream work. Destinations are
// checked (aligned, disjoint, reachable by the device) before anything is
// enqueued.
#include <hip/hip_runtime.h>

#include <fcntl.h>

#include <algorithm>
#include <cerrno>
#include <cmath>
#include <cstring>
#include <memory>
#include <mutex>
#include <vector>

#include "copy_pool.h"
#include "ii_internal.h"
#include "pertensor.h"
#include "reach.h"

namespace ii {

hipError_t launch_scatter_slot(const uint8_t* slot, const TileDev* tiles, const TileWin* wins,
                               uint32_t ntiles, const SegDev* segs, bool implicit,
                               uint32_t tile_bytes, uint64_t plen, hipStream_t stream);
hipError_t launch_scatter_layout(const uint8_t* span, const TileDev* tiles, const uint32_t* win,
                                 uint64_t ntiles, const LayoutSeg* segs, uint32_t tile_bytes,
                                 bool mixed, hipStream_t stream);
hipError_t launch_zero(const RangeDev* ranges, uint32_t n, hipStream_t stream);

#define II_HIP(call)                                                                   \
    do {                                                                               \
        hipError_t e_ = (call);                                                        \
        if (e_ != hipSuccess) {                                                        \
            (void)hipGetLastError();                                                   \
            return fail(e_ == hipErrorOutOfMemory ? II_ENOMEM : II_EHIP, "%s: %s (%s:%d)", \
                        #call, hipGetErrorString(e_), __FILE__, __LINE__);             \
        }                                                                              \
    } while (0)

// ---------------------------------------------------------------------------
// Failure injection, for tests of the error contract: with
// $II_TEST_FAIL_AT = "<site>:<n>" the n-th HIP call of one kind within one
// entry-point call returns an error instead of being made -- host_alloc
// (pinned host allocations), dev_alloc (device allocations), h2d
// (host-to-device copies and uploads), launch (kernel launches). Nothing is
// enqueued for the failing call, so the device sees no fault; the call then
// unwinds exactly as after a real runtime error.
enum InjectSite { kSiteHostAlloc, kSiteDevAlloc, kSiteH2D, kSiteLaunch, kNumSites };

struct Inject {
    int site = -1;
    long at = 0, seen = 0;
};
static thread_local Inject g_inject;

// Read $II_TEST_FAIL_AT at the entry of a call; counts restart from zero.
static void inject_arm() {
    static const char* const names[kNumSites] = {"host_alloc", "dev_alloc", "h2d", "launch"};
    g_inject = Inject{};
    const char* s = getenv("II_TEST_FAIL_AT");
    const char* colon = s ? strchr(s, ':') : nullptr;
    if (!colon) return;
    const long n = strtol(colon + 1, nullptr, 10);
    for (int i = 0; i < kNumSites; ++i)
        if ((size_t)(colon - s) == strlen(names[i]) && !strncmp(s, names[i], colon - s) && n > 0)
            g_inject = Inject{i, n, 0};
}

static bool injected(int site) { return g_inject.site == site && ++g_inject.seen == g_inject.at; }

template <class T>
static hipError_t dev_alloc(T** p, size_t n) {
    return injected(kSiteDevAlloc) ? hipErrorOutOfMemory
                                   : hipMalloc(reinterpret_cast<void**>(p), n);
}
template <class T>
static hipError_t host_alloc(T** p, size_t n) {
    return injected(kSiteHostAlloc) ? hipErrorOutOfMemory
                                    : hipHostMalloc(reinterpret_cast<void**>(p), n, 0);
}
static hipError_t h2d(void* d, const void* s, size_t n, hipStream_t st) {
    return injected(kSiteH2D) ? hipErrorUnknown
                              : hipMemcpyAsync(d, s, n, hipMemcpyHostToDevice, st);
}
static hipError_t h2d_2d(void* d, size_t dpitch, const void* s, size_t spitch, size_t w,
                         size_t h, hipStream_t st) {
    return injected(kSiteH2D) ? hipErrorUnknown
                              : hipMemcpy2DAsync(d, dpitch, s, spitch, w, h,
                                                 hipMemcpyHostToDevice, st);
}
static hipError_t h2d_sync(void* d, const void* s, size_t n) {
    return injected(kSiteH2D) ? hipErrorUnknown : hipMemcpy(d, s, n, hipMemcpyHostToDevice);
}
static bool launch_injected() { return injected(kSiteLaunch); }

struct Runtime {
    int device = -1;
    // device tables of the ring: segment rows with chunk offsets, tiles and
    // (plans with gaps) their windows
    SegDev* d_segs = nullptr;
    SegDev* h_segs = nullptr;  // pinned staging for d_segs uploads
    TileDev* d_tiles = nullptr;
    TileWin* d_wins = nullptr;
    // segment rows with packed staging offsets (plans with packed_distinct)
    SegDev* d_psegs = nullptr;
    SegDev* h_psegs = nullptr;
    bool tiles_ready = false, wins_ready = false;  // uploaded
    // device tables of the resident-image kernel: layout-order rows, layout
    // tiles and (layouts with padding-only windows) their windows
    LayoutSeg* d_lsegs = nullptr;
    LayoutSeg* h_lsegs = nullptr;  // pinned staging for d_lsegs uploads
    TileDev* d_ltiles = nullptr;
    uint32_t* d_lwin = nullptr;
    bool ltiles_ready = false, lwin_ready = false;  // uploaded
    hipEvent_t tables_idle = nullptr;   // after the last kernel that read a row table
    hipEvent_t upload_done = nullptr;   // after the last read of h_segs / h_psegs / h_lsegs
    bool tables_used = false, uploaded = false;
    std::vector<uint64_t> cached_dst;   // destination addresses of the last load
    std::vector<DstRange> cached_ranges;  // ... their ranges, sorted by address
    bool cached_valid = false;
    // whether d_segs (and d_psegs) / d_lsegs hold rows for cached_dst
    bool ring_rows_ok = false, layout_rows_ok = false;
    uint64_t image_b = 0, image_e = 0;  // source image range last checked against them
    // scrub ranges
    RangeDev* d_ranges = nullptr;
    RangeDev* h_ranges = nullptr;
    size_t ranges_cap = 0;
    hipEvent_t ranges_idle = nullptr;
    bool ranges_used = false;
    // ring
    uint32_t depth = 0;
    std::vector<uint8_t*> hslot, dslot;
    std::vector<hipEvent_t> copy_done, scatter_done;
    std::vector<char> copy_rec, scatter_rec;
    std::vector<int> slot_lane;  // lane of the last scatter that read each device slot (-1: none)
    // lanes: chunk j's copy and then its scatter run on lane j mod nlanes
    hipStream_t lane_s[kMaxLanes] = {};
    hipEvent_t lane_done[kMaxLanes] = {};
    uint32_t nlanes = 1;
    hipEvent_t entry = nullptr, go = nullptr, done = nullptr;
    CopyPool* pool = nullptr;
    // optional per-chunk timeline of the last ring load (timing events)
    std::vector<hipEvent_t> tr_cs, tr_ce, tr_ss, tr_se;
    hipEvent_t tr_t0 = nullptr;
    size_t tr_chunks = 0;          // chunks recorded by the last traced load (0 = none)
    std::vector<uint32_t> tr_id;   // chunk index of each recorded entry
    // chunks that hold at least one segment, in order (the ring skips the rest)
    std::vector<uint32_t> live;
    bool live_ready = false;
};

static void free_trace(Runtime* r) {
    for (auto* v : {&r->tr_cs, &r->tr_ce, &r->tr_ss, &r->tr_se}) {
        for (auto e : *v)
            if (e) (void)hipEventDestroy(e);
        v->clear();
    }
    if (r->tr_t0) (void)hipEventDestroy(r->tr_t0);
    r->tr_t0 = nullptr;
    r->tr_chunks = 0;
}

// ---------------------------------------------------------------------------
// state management

static void free_ring(Runtime* r) {
    for (auto p : r->hslot) if (p) (void)hipHostFree(p);
    for (auto p : r->dslot) if (p) (void)hipFree(p);
    for (auto e : r->copy_done) if (e) (void)hipEventDestroy(e);
    for (auto e : r->scatter_done) if (e) (void)hipEventDestroy(e);
    r->hslot.clear();
    r->dslot.clear();
    r->copy_done.clear();
    r->scatter_done.clear();
    r->copy_rec.clear();
    r->scatter_rec.clear();
    r->slot_lane.clear();
    for (auto& c : r->lane_s) {
        if (c) (void)hipStreamDestroy(c);
        c = nullptr;
    }
    for (auto& e : r->lane_done) {
        if (e) (void)hipEventDestroy(e);
        e = nullptr;
    }
    for (hipEvent_t* e : {&r->entry, &r->go, &r->done}) {
        if (*e) (void)hipEventDestroy(*e);
        *e = nullptr;
    }
    delete r->pool;
    r->pool = nullptr;
    r->depth = 0;
}

static void destroy(Runtime* r) {
    if (!r) return;
    int cur = -1;
    (void)hipGetDevice(&cur);
    if (r->device >= 0 && cur != r->device) (void)hipSetDevice(r->device);
    // drain everything the plan may still have in flight
    for (auto c : r->lane_s)
        if (c) (void)hipStreamSynchronize(c);
    if (r->tables_idle && r->tables_used) (void)hipEventSynchronize(r->tables_idle);
    if (r->upload_done && r->uploaded) (void)hipEventSynchronize(r->upload_done);
    if (r->ranges_idle && r->ranges_used) (void)hipEventSynchronize(r->ranges_idle);
    free_ring(r);
    free_trace(r);
    if (r->d_segs) (void)hipFree(r->d_segs);
    if (r->h_segs) (void)hipHostFree(r->h_segs);
    if (r->d_tiles) (void)hipFree(r->d_tiles);
    if (r->d_wins) (void)hipFree(r->d_wins);
    if (r->d_lsegs) (void)hipFree(r->d_lsegs);
    if (r->h_lsegs) (void)hipHostFree(r->h_lsegs);
    if (r->d_ltiles) (void)hipFree(r->d_ltiles);
    if (r->d_lwin) (void)hipFree(r->d_lwin);
    if (r->d_psegs) (void)hipFree(r->d_psegs);
    if (r->h_psegs) (void)hipHostFree(r->h_psegs);
    if (r->d_ranges) (void)hipFree(r->d_ranges);
    if (r->h_ranges) (void)hipHostFree(r->h_ranges);
    if (r->tables_idle) (void)hipEventDestroy(r->tables_idle);
    if (r->upload_done) (void)hipEventDestroy(r->upload_done);
    if (r->ranges_idle) (void)hipEventDestroy(r->ranges_idle);
    (void)hipGetLastError();
    if (r->device >= 0 && cur >= 0 && cur != r->device) (void)hipSetDevice(cur);
    delete r;
}

void runtime_destroy(ii_plan_t* p) {
    destroy(p->rt);
    p->rt = nullptr;
}

// The plan's device state, its events and its list of chunks that hold
// segments (the tables of either path come from ensure_ring_tables and
// ensure_layout_tables).
static int ensure_state(ii_plan_t* p) {
    int dev = -1;
    II_HIP(hipGetDevice(&dev));
    if (!p->rt) {
        p->rt = new (std::nothrow) Runtime();
        if (!p->rt) return fail(II_ENOMEM, "runtime state allocation failed");
        p->rt->device = dev;
    }
    Runtime* r = p->rt;
    if (r->device != dev)
        return fail(II_EINVAL, "plan was first used on device %d, current device is %d",
                    r->device, dev);
    for (hipEvent_t* e : {&r->tables_idle, &r->upload_done, &r->ranges_idle})
        if (!*e) II_HIP(hipEventCreateWithFlags(e, hipEventDisableTiming));
    if (!r->live_ready) {
        r->live.clear();
        for (size_t k = 0; k < p->num_chunks; ++k)
            if (p->chunk_seg_begin[k] < p->chunk_seg_begin[k + 1]) r->live.push_back((uint32_t)k);
        r->live_ready = true;
    }
    return II_OK;
}

// Each table is allocated and uploaded separately, and counted as ready only
// once its upload returned: a call that failed half-way (one allocation
// made, the next refused) leaves nothing a later load would take for
// initialised. The tile tables never change after they are uploaded
// (synchronously, once per plan).
static int ensure_ring_tables(ii_plan_t* p) {
    Runtime* r = p->rt;
    const size_t S = p->seg_len.size();
    if (S && !r->d_segs) II_HIP(dev_alloc(&r->d_segs, S * sizeof(SegDev)));
    if (S && !r->h_segs) II_HIP(host_alloc(&r->h_segs, S * sizeof(SegDev)));
    if (S && p->packed_distinct) {
        if (!r->d_psegs) II_HIP(dev_alloc(&r->d_psegs, S * sizeof(SegDev)));
        if (!r->h_psegs) II_HIP(host_alloc(&r->h_psegs, S * sizeof(SegDev)));
    }
    if (!p->tile_win.empty() && !r->wins_ready) {
        if (!r->d_wins) II_HIP(dev_alloc(&r->d_wins, p->tile_win.size() * sizeof(TileWin)));
        II_HIP(h2d_sync(r->d_wins, p->tile_win.data(), p->tile_win.size() * sizeof(TileWin)));
        r->wins_ready = true;
    }
    if (!p->tiles.empty() && !r->tiles_ready) {
        if (!r->d_tiles) II_HIP(dev_alloc(&r->d_tiles, p->tiles.size() * sizeof(TileDev)));
        II_HIP(h2d_sync(r->d_tiles, p->tiles.data(), p->tiles.size() * sizeof(TileDev)));
        r->tiles_ready = true;
    }
    return II_OK;
}

static int ensure_layout_tables(ii_plan_t* p) {
    Runtime* r = p->rt;
    const size_t S = p->seg_len.size();
    if (S && !r->d_lsegs) II_HIP(dev_alloc(&r->d_lsegs, S * sizeof(LayoutSeg)));
    if (S && !r->h_lsegs) II_HIP(host_alloc(&r->h_lsegs, S * sizeof(LayoutSeg)));
    if (!p->lwin.empty() && !r->lwin_ready) {
        if (!r->d_lwin) II_HIP(dev_alloc(&r->d_lwin, p->lwin.size() * sizeof(uint32_t)));
        II_HIP(h2d_sync(r->d_lwin, p->lwin.data(), p->lwin.size() * sizeof(uint32_t)));
        r->lwin_ready = true;
    }
    if (!p->ltiles.empty() && !r->ltiles_ready) {
        if (!r->d_ltiles) II_HIP(dev_alloc(&r->d_ltiles, p->ltiles.size() * sizeof(TileDev)));
        II_HIP(h2d_sync(r->d_ltiles, p->ltiles.data(), p->ltiles.size() * sizeof(TileDev)));
        r->ltiles_ready = true;
    }
    return II_OK;
}

static int ensure_ring(ii_plan_t* p) {
    Runtime* r = p->rt;
    if (r->depth) return II_OK;
    const uint32_t D = p->ring_depth;
    r->hslot.assign(D, nullptr);
    r->dslot.assign(D, nullptr);
    r->copy_done.assign(D, nullptr);
    r->scatter_done.assign(D, nullptr);
    r->copy_rec.assign(D, 0);
    r->scatter_rec.assign(D, 0);
    r->slot_lane.assign(D, -1);
    r->depth = D;  // free_ring() cleans up partial state on failure below
    int rc = II_OK;
    auto bail = [&](int code) {
        free_ring(r);
        return code;
    };
#define II_RING(call)                                                                    \
    do {                                                                                 \
        rc = [&]() -> int { II_HIP(call); return II_OK; }();                             \
        if (rc) return bail(rc);                                                         \
    } while (0)
    const uint64_t C = p->chunk_bytes;
    for (uint32_t i = 0; i < D; ++i) {
        II_RING(host_alloc(&r->hslot[i], C));
        II_RING(dev_alloc(&r->dslot[i], C));
        II_RING(hipEventCreateWithFlags(&r->copy_done[i], hipEventDisableTiming));
        II_RING(hipEventCreateWithFlags(&r->scatter_done[i], hipEventDisableTiming));
    }
    r->nlanes = p->copy_streams;
    for (uint32_t i = 0; i < r->nlanes; ++i) {
        II_RING(hipStreamCreateWithFlags(&r->lane_s[i], hipStreamNonBlocking));
        II_RING(hipEventCreateWithFlags(&r->lane_done[i], hipEventDisableTiming));
    }
    II_RING(hipEventCreateWithFlags(&r->entry, hipEventDisableTiming));
    II_RING(hipEventCreateWithFlags(&r->go, hipEventDisableTiming));
    II_RING(hipEventCreateWithFlags(&r->done, hipEventDisableTiming));
#undef II_RING
    r->pool = new (std::nothrow) CopyPool(p->host_threads);
    if (!r->pool) return bail(fail(II_ENOMEM, "host copy pool allocation failed"));
    for (uint32_t i = 0; i < D; ++i) r->pool->touch(r->hslot[i], C);
    return II_OK;
}

// Timing events for a traced load of K chunks.
static int ensure_trace(Runtime* r, size_t K) {
    if (r->tr_cs.size() >= K && r->tr_t0) return II_OK;
    free_trace(r);
    for (auto* v : {&r->tr_cs, &r->tr_ce, &r->tr_ss, &r->tr_se}) {
        v->assign(K, nullptr);
        for (auto& e : *v) II_HIP(hipEventCreate(&e));
    }
    II_HIP(hipEventCreate(&r->tr_t0));
    return II_OK;
}

// ---------------------------------------------------------------------------
// argument checks

// What HIP reports about the allocation holding address x.
static AllocInfo alloc_info(uint64_t x) {
    AllocInfo info;
    hipPointerAttribute_t a;
    if (hipPointerGetAttributes(&a, reinterpret_cast<void*>(x)) != hipSuccess) {
        (void)hipGetLastError();
        return info;
    }
    if (a.type == hipMemoryTypeDevice || a.type == hipMemoryTypeManaged)
        info.kind = AllocInfo::kDevice;
    else if (a.type == hipMemoryTypeHost)
        info.kind = AllocInfo::kPinnedHost;
    else
        return info;
    hipDeviceptr_t base = nullptr;
    size_t size = 0;
    if (hipMemGetAddressRange(&base, &size, reinterpret_cast<hipDeviceptr_t>(x)) != hipSuccess) {
        (void)hipGetLastError();
        return info;
    }
    info.extent = true;
    info.base = reinterpret_cast<uint64_t>(base);
    info.size = size;
    return info;
}

// Whether the device can reach [b, e): the whole range inside one device
// allocation or one pinned host allocation (reach.h). A kernel or a DMA
// touching pageable memory, unknown memory, or a range that runs from one
// allocation into whatever lies past its end would fault the device.
static bool accessible(uint64_t b, uint64_t e) { return reachable(alloc_info(b), b, e); }

// Destination ranges of the non-empty tensors, sorted by address, after
// checking that each is present, aligned and disjoint from the others.
static int dst_ranges(const ii_plan_t* p, const uint64_t* dst, std::vector<DstRange>* out) {
    const size_t n = p->nbytes.size();
    std::vector<DstRange>& v = *out;
    v.clear();
    v.reserve(n);
    for (size_t i = 0; i < n; ++i) {
        if (!p->nbytes[i]) continue;
        if (!dst[i]) return fail(II_EINVAL, "dst_ptrs[%zu] is NULL for a non-empty tensor", i);
        if (dst[i] & (p->dst_align[i] - 1))
            return fail(II_EALIGN, "dst_ptrs[%zu]=%#llx is not aligned to %llu", i,
                        (unsigned long long)dst[i], (unsigned long long)p->dst_align[i]);
        uint64_t e;
        if (__builtin_add_overflow(dst[i], p->nbytes[i], &e))
            return fail(II_EOVERFLOW, "dst_ptrs[%zu] + nbytes overflows", i);
        v.push_back({dst[i], e, i});
    }
    std::sort(v.begin(), v.end(), [](const DstRange& a, const DstRange& b) { return a.b < b.b; });
    for (size_t j = 1; j < v.size(); ++j)
        if (v[j].b < v[j - 1].e)
            return fail(II_EOVERLAP, "destinations of tensors %zu and %zu overlap", v[j - 1].i,
                        v[j].i);
    return II_OK;
}

// Every range (sorted by address) reachable by the device: one allocation
// query per allocation the ranges fall in.
static int check_reach(const std::vector<DstRange>& v) {
    const size_t j = first_unreachable(v, alloc_info);
    if (j == v.size()) return II_OK;
    return fail(II_EINVAL, "dst_ptrs[%zu]=%#llx (+%llu bytes) is not memory the device can "
                "write: not inside one device allocation or one pinned host allocation",
                v[j].i, (unsigned long long)v[j].b, (unsigned long long)(v[j].e - v[j].b));
}

// Check destination addresses: present, aligned, pairwise disjoint and
// reachable by the device.
static int check_dst(const ii_plan_t* p, const uint64_t* dst) {
    std::vector<DstRange> v;
    int rc = dst_ranges(p, dst, &v);
    return rc ? rc : check_reach(v);
}

// No destination may overlap the source image [b, e) (one linear pass).
static int check_image(const ii_plan_t* p, const uint64_t* dst, uint64_t b, uint64_t e) {
    for (size_t i = 0; i < p->nbytes.size(); ++i)
        if (p->nbytes[i] && dst[i] < e && b < dst[i] + p->nbytes[i])
            return fail(II_EOVERLAP, "tensor %zu's destination overlaps the source image", i);
    return II_OK;
}

// Make the row tables a load reads (`which`: the ring's, the resident-image
// kernel's) hold its resolved destination addresses. The upload is ordered
// on `s`, after every kernel that read the previous tables. The
// checks that depend only on the addresses (present, aligned, disjoint) run
// for destinations not seen before; reachability -- whether the memory is
// still allocated -- is checked on every call, one query per allocation,
// since a freed arena may be passed again at the same addresses.
enum RowTables { kRingRows = 1, kLayoutRows = 2 };

static int prepare_segments(ii_plan_t* p, const uint64_t* dst, hipStream_t s, uint64_t image_b,
                            uint64_t image_e, int which) {
    Runtime* r = p->rt;
    const size_t n = p->nbytes.size(), S = p->seg_len.size();
    const bool same = r->cached_valid && r->cached_dst.size() == n &&
                      (n == 0 || memcmp(r->cached_dst.data(), dst, n * sizeof(uint64_t)) == 0);
    if (!same) {
        r->cached_valid = false;
        try {
            int rc = dst_ranges(p, dst, &r->cached_ranges);
            if (rc) return rc;
        } catch (const std::bad_alloc&) {
            return fail(II_ENOMEM, "destination check: host allocation failed");
        }
    }
    int rc = check_reach(r->cached_ranges);
    if (rc) return rc;
    if (image_e > image_b) {
        if (!accessible(image_b, image_e))
            return fail(II_EINVAL, "the image's span [%#llx, %#llx) is not memory the device can "
                        "read: not inside one device allocation or one pinned host allocation",
                        (unsigned long long)image_b, (unsigned long long)image_e);
        if (!(same && r->image_b == image_b && r->image_e == image_e)) {
            rc = check_image(p, dst, image_b, image_e);
            if (rc) return rc;
        }
    }
    if (!same) {
        // new destinations: every row table is stale until rebuilt for them
        r->ring_rows_ok = r->layout_rows_ok = false;
        try {
            r->cached_dst.assign(dst, dst + n);
        } catch (const std::bad_alloc&) {
            return fail(II_ENOMEM, "destination check: host allocation failed");
        }
        r->cached_valid = true;
    }
    r->image_b = image_b;
    r->image_e = image_e;
    const bool ring = S && (which & kRingRows) && !r->ring_rows_ok;
    const bool layout = S && (which & kLayoutRows) && !r->layout_rows_ok;
    if (!ring && !layout) return II_OK;
    if (r->uploaded) II_HIP(hipEventSynchronize(r->upload_done));  // staging buffers free again
    if (ring) {
        for (size_t i = 0; i < S; ++i)
            r->h_segs[i] = SegDev{p->seg_off[i], p->seg_len[i],
                                  dst[p->seg_tensor[i]] + p->seg_toff[i]};
        if (p->packed_distinct)
            for (size_t i = 0; i < S; ++i)
                r->h_psegs[i] = SegDev{p->seg_poff[i], p->seg_len[i], r->h_segs[i].dst};
    }
    if (layout) {
        const uint64_t C = p->chunk_bytes;
        for (size_t j = 0; j < S; ++j) {
            const uint32_t x = p->lseg[j], t = p->seg_tensor[x];
            r->h_lsegs[j] = LayoutSeg{(uint64_t)p->seg_chunk[x] * C + p->seg_off[x],
                                      dst[t] + p->seg_toff[x], p->dst_offset[t] + p->seg_toff[x],
                                      p->seg_len[x], 0};
        }
    }
    if (r->tables_used) II_HIP(hipStreamWaitEvent(s, r->tables_idle, 0));
    if (ring) {
        II_HIP(h2d(r->d_segs, r->h_segs, S * sizeof(SegDev), s));
        if (p->packed_distinct) II_HIP(h2d(r->d_psegs, r->h_psegs, S * sizeof(SegDev), s));
    }
    if (layout) II_HIP(h2d(r->d_lsegs, r->h_lsegs, S * sizeof(LayoutSeg), s));
    II_HIP(hipEventRecord(r->upload_done, s));
    r->uploaded = true;
    if (ring) r->ring_rows_ok = true;
    if (layout) r->layout_rows_ok = true;
    return II_OK;
}

// Upload the scrub ranges and launch the zero fill on `s`.
static int launch_scrub(ii_plan_t* p, const std::vector<RangeDev>& ranges, hipStream_t s) {
    Runtime* r = p->rt;
    if (ranges.empty()) return II_OK;
    if (ranges.size() > 0x7fffffffull) return fail(II_EINVAL, "too many scrub ranges");
    if (r->ranges_used) II_HIP(hipEventSynchronize(r->ranges_idle));
    if (ranges.size() > r->ranges_cap) {
        if (r->d_ranges) II_HIP(hipFree(r->d_ranges));
        if (r->h_ranges) II_HIP(hipHostFree(r->h_ranges));
        r->d_ranges = nullptr;
        r->h_ranges = nullptr;
        r->ranges_cap = 0;
        II_HIP(dev_alloc(&r->d_ranges, ranges.size() * sizeof(RangeDev)));
        II_HIP(host_alloc(&r->h_ranges, ranges.size() * sizeof(RangeDev)));
        r->ranges_cap = ranges.size();
    }
    memcpy(r->h_ranges, ranges.data(), ranges.size() * sizeof(RangeDev));
    II_HIP(h2d(r->d_ranges, r->h_ranges, ranges.size() * sizeof(RangeDev), s));
    II_HIP(launch_injected() ? hipErrorLaunchFailure
                             : launch_zero(r->d_ranges, (uint32_t)ranges.size(), s));
    II_HIP(hipEventRecord(r->ranges_idle, s));
    r->ranges_used = true;
    return II_OK;
}

// Whether the blob bytes a load reads, [blob + lo, blob + hi), lie inside one
// pinned host allocation, so that copies may read them by DMA. A blob pinned
// only in part (or whose span reaches past its pinned allocation) is treated
// as pageable: the host stage copies it, and no DMA reads outside pinned
// memory.
static bool pinned_span(const ii_plan_t* p, const uint8_t* blob) {
    if (p->hi <= p->lo) return false;
    const uint64_t b = reinterpret_cast<uint64_t>(blob) + p->lo;
    const uint64_t e = reinterpret_cast<uint64_t>(blob) + p->hi;
    const AllocInfo a = alloc_info(b);
    return a.kind == AllocInfo::kPinnedHost && reachable(a, b, e);
}

static bool is_device_ptr(const void* ptr) {
    hipPointerAttribute_t a;
    hipError_t e = hipPointerGetAttributes(&a, ptr);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return false;
    }
    return a.type == hipMemoryTypeDevice;
}

// Drain the plan's streams after an error so that nothing enqueued by the
// failed call still touches caller memory.
static int drain(ii_plan_t* p, hipStream_t caller, int rc) {
    if (p->rt)
        for (auto c : p->rt->lane_s)
            if (c) (void)hipStreamSynchronize(c);
    (void)hipStreamSynchronize(caller);
    (void)hipGetLastError();
    return rc;
}

struct BusyGuard {
    ii_plan_t* p;
    bool ok;
    explicit BusyGuard(ii_plan_t* q) : p(q) {
        int expect = 0;
        ok = p->busy.compare_exchange_strong(expect, 1);
    }
    ~BusyGuard() {
        if (ok) p->busy.store(0);
    }
};

// ---------------------------------------------------------------------------
// the pipeline

// Where the chunk bytes come from: a host blob (pageable: copied into the
// pinned slot by the host threads; pinned: copied by DMA straight from it) or
// a file (read into the pinned slot by the host threads; with O_DIRECT the
// reads start and end on kIoAlign boundaries and the chunk sits `shift`
// bytes into the slot).
struct Source {
    const uint8_t* blob = nullptr;
    int fd = -1;
    bool direct = false;
};

static int run_ring(ii_plan_t* p, const Source& src, const uint64_t* dst, hipStream_t stream,
                    const std::vector<RangeDev>* scrub) {
    int rc = ensure_state(p);
    if (rc) return rc;
    rc = ensure_ring_tables(p);
    if (rc) return rc;
    rc = ensure_ring(p);
    if (rc) return rc;
    Runtime* r = p->rt;
    const uint8_t* blob = src.blob;
    const bool pinned = src.fd < 0 && pinned_span(p, blob);
    // The host stage gathers packed chunks whenever it copies anyway, and
    // for a pinned blob also where most of a chunk's used range is gaps.

    const bool trace = p->trace;
    if (trace) {
        rc = ensure_trace(r, p->num_chunks);
        if (rc) return rc;
        r->tr_chunks = 0;
    }
    // Destination checks; new destinations' rows are uploaded on lane 0,
    // ahead of every scatter of this load.
    hipStream_t lane0 = r->lane_s[0];
    rc = prepare_segments(p, dst, lane0, 0, 0, kRingRows);
    if (rc) return rc;
    // Entry edge: destination writes start after the caller's prior work.
    // Copies into the ring need no such wait (they write only the plan's own
    // slots), so each lane's first copy may run while that work is still
    // pending; the lane waits before its first scatter. Lane 0 opens first
    // (chunk 0 is its): it waits for the entry event, runs the scrub of a
    // switch, and records `go`; every other lane waits for `go`.
    II_HIP(hipEventRecord(r->entry, stream));
    uint32_t opened = 0;  // bit l: lane l's scatters are ordered after `go`
    auto open_lane = [&](uint32_t l) -> int {
        if (opened & (1u << l)) return II_OK;
        if (!(opened & 1u)) {
            II_HIP(hipStreamWaitEvent(lane0, r->entry, 0));
            if (trace) II_HIP(hipEventRecord(r->tr_t0, lane0));
            if (scrub) {
                const int e = launch_scrub(p, *scrub, lane0);
                if (e) return e;
            }
            II_HIP(hipEventRecord(r->go, lane0));
            opened |= 1u;
        }
        if (l) II_HIP(hipStreamWaitEvent(r->lane_s[l], r->go, 0));
        opened |= 1u << l;
        return II_OK;
    };

    const uint32_t D = r->depth;
    const uint64_t C = p->chunk_bytes;
    // Chunk j of the ring is chunk live[j] of the plan. Packed: the host
    // stage gathers the chunk's segments back to back and only they cross
    // the link. Otherwise (pinned blob) the used range [u0, u1) of the chunk
    // crosses at its own offsets in the slot.
    const std::vector<uint32_t>& live = r->live;
    const uint32_t L = (uint32_t)live.size();
    std::unique_ptr<ReadAhead> ahead;
    if (src.fd >= 0 && src.direct && L) {
        const uint64_t lo = p->lo;
        try {
            ahead.reset(new ReadAhead(
            src.fd, std::min<uint32_t>(p->host_threads, 8), C + 2 * kIoAlign, L,
            [p, lo, C, &live](uint32_t j) {
                uint64_t u0, u1;
                p->chunk_used(live[j], &u0, &u1);
                const uint64_t at = lo + (uint64_t)live[j] * C + u0, len = u1 - u0;
                const uint64_t a = at & ~(kIoAlign - 1);
                const uint64_t e = (at + len + kIoAlign - 1) & ~(kIoAlign - 1);
                return ReadAhead::Range{a, e, at + len - a};
            }));
        } catch (const std::exception&) {
            return fail(II_ENOMEM, "read-ahead threads could not be started");
        }
        if (!ahead->ok()) return fail(II_ENOMEM, "read-ahead buffer allocation failed");
    }
    for (uint32_t j = 0; j < L; ++j) {
        const uint32_t k = live[j], slot = j % D;
        uint64_t u0, u1;
        p->chunk_used(k, &u0, &u1);
        const uint64_t cbeg = p->lo + (uint64_t)k * C;  // blob / file offset of the chunk
        const uint64_t at = cbeg + u0;                   // ... and of its used range
        // a pinned blob's chunk of a plan with gaps: moved in place, by
        // copies of its run groups, or gathered on the host
        const uint8_t how = pinned && p->packed_distinct ? p->chunk_pinned[k] : kPinnedInPlace;
        const bool packed = p->packed_distinct && (!pinned || how != kPinnedInPlace);
        const bool staged = !pinned || how == kPinnedGather;  // through the pinned slot
        // packed: the slot receives the chunk's runs back to back from offset
        // 0; otherwise the used range keeps its chunk offsets
        const uint64_t r0 = p->chunk_run_begin[k], nr = p->chunk_run_begin[k + 1] - r0;
        const uint64_t len = packed ? p->chunk_plen[k] : u1 - u0;
        const uint64_t doff = packed ? 0 : u0;
        const uint8_t* from = blob ? blob + at : nullptr;
        // InMem -> InGPU on lane l, once the device slot's previous scatter
        // is done (implied when that scatter ran on this lane)
        const uint32_t l = j % r->nlanes;
        hipStream_t cs = r->lane_s[l];
        if (staged) {
            // InDisk -> InMem: the pinned slot is free once its last copy finished
            if (r->copy_rec[slot]) II_HIP(hipEventSynchronize(r->copy_done[slot]));
            uint8_t* stage = r->hslot[slot] + doff;
            const uint32_t *ro = p->run_off.data() + r0, *rp = p->run_poff.data() + r0,
                           *rl = p->run_len.data() + r0;
            if (src.fd < 0) {
                if (packed) r->pool->gather(stage, blob + cbeg, 0, ro, rp, rl, nr, len);
                else r->pool->copy(stage, from, len);
            } else if (!src.direct) {
                const int err = packed ? r->pool->read_gather(src.fd, stage, cbeg, ro, rp, rl, nr, len)
                                       : r->pool->read(src.fd, stage, at, len, 1, len);
                if (err)
                    return fail(II_EIO, "reading chunk %u (file bytes %llu..%llu): %s", k,
                                (unsigned long long)at, (unsigned long long)(cbeg + u1),
                                strerror(err));
            } else {
                // direct I/O: whole blocks, read ahead into aligned buffers;
                // the chunk's bytes are then copied into the pinned slot
                int err = 0;
                const uint8_t* b = ahead->wait(j, &err);
                if (!b)
                    return fail(II_EIO, "reading chunk %u (file bytes from %llu): %s", k,
                                (unsigned long long)(at & ~(kIoAlign - 1)), strerror(err));
                const uint64_t a = at & ~(kIoAlign - 1);  // file offset of b[0]
                if (packed)  // b[0] is chunk offset a - cbeg (may be negative)
                    r->pool->gather(stage, b, (int64_t)(a - cbeg), ro, rp, rl, nr, len);
                else
                    r->pool->copy(stage, b + (at - a), len);
                ahead->release(j);
            }
            from = stage;
        }
        if (r->scatter_rec[slot] && r->slot_lane[slot] != (int)l)
            II_HIP(hipStreamWaitEvent(cs, r->scatter_done[slot], 0));
        if (trace) II_HIP(hipEventRecord(r->tr_cs[j], cs));
        if (pinned && how == kPinnedGroups) {
            // one copy per run group straight from the pinned blob into the
            // packed layout: rows of a group land back to back
            for (uint64_t gi = p->chunk_group_begin[k]; gi < p->chunk_group_begin[k + 1]; ++gi) {
                const DmaGroup& g = p->groups[gi];
                uint8_t* to = r->dslot[slot] + g.poff;
                const uint8_t* at = blob + cbeg + g.off;
                if (g.count == 1)
                    II_HIP(h2d(to, at, g.len, cs));
                else
                    II_HIP(h2d_2d(to, g.len, at, g.stride, g.len, g.count, cs));
            }
        } else {
            II_HIP(h2d(r->dslot[slot] + doff, from, len, cs));
        }
        II_HIP(hipEventRecord(r->copy_done[slot], cs));
        if (trace) II_HIP(hipEventRecord(r->tr_ce[j], cs));
        r->copy_rec[slot] = 1;
        // InGPU -> tensors Loaded on the same lane, after the copy; then the
        // slot is released
        rc = open_lane(l);
        if (rc) return rc;
        if (trace) II_HIP(hipEventRecord(r->tr_ss[j], cs));
        const uint64_t t0 = p->chunk_tile_begin[k], nt = p->chunk_tile_begin[k + 1] - t0;
        // windows are implicit in a packed slot and in a plan without gaps
        // (which keeps no window table)
        const bool implicit = packed || !p->packed_distinct;
        II_HIP(launch_injected() ? hipErrorLaunchFailure
                                 : launch_scatter_slot(r->dslot[slot], r->d_tiles + t0,
                                   implicit ? nullptr : r->d_wins + t0, (uint32_t)nt,
                                   packed ? r->d_psegs : r->d_segs, implicit, p->tile_bytes,
                                   p->chunk_plen[k], cs));
        II_HIP(hipEventRecord(r->scatter_done[slot], cs));
        if (trace) II_HIP(hipEventRecord(r->tr_se[j], cs));
        r->scatter_rec[slot] = 1;
        r->slot_lane[slot] = (int)l;
    }
    if (trace) {
        r->tr_id = live;
        r->tr_chunks = L;
    }
    // a load without chunks still waits for the entry edge and runs the scrub
    rc = open_lane(0);
    if (rc) return rc;
    // completion: lane 0 joins the other lanes, the caller's stream waits
    for (uint32_t x = 1; x < r->nlanes; ++x)
        if (opened & (1u << x)) {
            II_HIP(hipEventRecord(r->lane_done[x], r->lane_s[x]));
            II_HIP(hipStreamWaitEvent(lane0, r->lane_done[x], 0));
        }
    II_HIP(hipEventRecord(r->tables_idle, lane0));
    r->tables_used = true;
    II_HIP(hipEventRecord(r->done, lane0));
    II_HIP(hipStreamWaitEvent(stream, r->done, 0));
    return II_OK;
}

static int run_device(ii_plan_t* p, const uint8_t* image, const uint64_t* dst, hipStream_t stream) {
    int rc = ensure_state(p);
    if (rc) return rc;
    rc = ensure_layout_tables(p);
    if (rc) return rc;
    Runtime* r = p->rt;
    const uint64_t ib = reinterpret_cast<uint64_t>(image);
    rc = prepare_segments(p, dst, stream, ib + p->lo, ib + p->hi, kLayoutRows);
    if (rc) return rc;
    II_HIP(launch_injected() ? hipErrorLaunchFailure
                             : launch_scatter_layout(image + p->lo, r->d_ltiles, r->d_lwin,
                                                     p->ltiles.size(), r->d_lsegs, p->tile_bytes,
                                                     p->layout_mixed, stream));
    II_HIP(hipEventRecord(r->tables_idle, stream));
    r->tables_used = true;
    return II_OK;
}

// ---------------------------------------------------------------------------
// The resident-image load without allocation: the kernel's tables go into
// `scratch`, a static device array each GPU holds for the life of the
// process, uploaded on the call's stream every time (another plan's call may
// have overwritten them in between).
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static uint8_t* g_scratch[kMaxDevices];  // device address of `scratch`, per device

// The device address of the current device's copy of `scratch`, looked up
// once per device. (In host code the array's name is only a host-side
// stand-in for the symbol; kernels and copies must use this address.)
static int scratch_ptr(uint8_t** out) {
    int dev = -1;
    II_HIP(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxDevices)
        return fail(II_EINVAL, "device %d is beyond the %d the library supports", dev, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[dev]) {
        void* ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !ptr) {
            (void)hipGetLastError();
            return fail(II_EHIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev,
                        hipGetErrorString(e));
        }
        g_scratch[dev] = static_cast<uint8_t*>(ptr);
    }
    *out = g_scratch[dev];
    return II_OK;
}

// Where each table of a plan sits in the workspace (offsets 256-aligned).
struct ScratchLayout {
    uint64_t rows, tiles, win, end;
};

static ScratchLayout scratch_layout(const ii_plan_t* p) {
    auto up = [](uint64_t x) { return (x + 255) & ~255ull; };
    ScratchLayout l;
    l.rows = 0;
    l.tiles = up(p->lseg.size() * sizeof(LayoutSeg));
    l.win = up(l.tiles + p->ltiles.size() * sizeof(TileDev));
    l.end = l.win + p->lwin.size() * sizeof(uint32_t);
    return l;
}

static int run_device_noalloc(ii_plan_t* p, const uint8_t* image, const uint64_t* dst,
                              hipStream_t stream) {
    // destination checks into the plan's own buffer (its capacity is the
    // table's size, so nothing is allocated)
    int rc = dst_ranges(p, dst, &p->na_ranges);
    if (rc) return rc;
    rc = check_reach(p->na_ranges);
    if (rc) return rc;
    if (p->ltiles.empty()) return II_OK;  // nothing to move
    const uint64_t ib = reinterpret_cast<uint64_t>(image);
    if (!accessible(ib + p->lo, ib + p->hi))
        return fail(II_EINVAL, "the image's span [%#llx, %#llx) is not memory the device can "
                    "read: not inside one device allocation or one pinned host allocation",
                    (unsigned long long)(ib + p->lo), (unsigned long long)(ib + p->hi));
    rc = check_image(p, dst, ib + p->lo, ib + p->hi);
    if (rc) return rc;
    uint8_t* ws = nullptr;
    rc = scratch_ptr(&ws);
    if (rc) return rc;
    const ScratchLayout l = scratch_layout(p);
    const size_t S = p->lseg.size();
    const uint64_t C = p->chunk_bytes;
    for (size_t j = 0; j < S; ++j) {
        const uint32_t x = p->lseg[j], t = p->seg_tensor[x];
        p->na_rows[j] = LayoutSeg{(uint64_t)p->seg_chunk[x] * C + p->seg_off[x],
                                  dst[t] + p->seg_toff[x], p->dst_offset[t] + p->seg_toff[x],
                                  p->seg_len[x], 0};
    }
    // pageable sources: each copy returns once its bytes are staged, so the
    // plan's buffers may be rewritten by the next call
    if (S) II_HIP(h2d(ws + l.rows, p->na_rows.data(), S * sizeof(LayoutSeg), stream));
    II_HIP(h2d(ws + l.tiles, p->ltiles.data(), p->ltiles.size() * sizeof(TileDev), stream));
    if (!p->lwin.empty())
        II_HIP(h2d(ws + l.win, p->lwin.data(), p->lwin.size() * sizeof(uint32_t), stream));
    II_HIP(launch_injected()
               ? hipErrorLaunchFailure
               : launch_scatter_layout(
                     image + p->lo, reinterpret_cast<const TileDev*>(ws + l.tiles),
                     p->lwin.empty() ? nullptr : reinterpret_cast<const uint32_t*>(ws + l.win),
                     p->ltiles.size(), reinterpret_cast<const LayoutSeg*>(ws + l.rows),
                     p->tile_bytes, p->layout_mixed, stream));
    return II_OK;
}

// The naive per-tensor pipeline of Sec. 4.2 ("Naive CFA Model"), kept as the
// comparison path for the merged loader: tensors in table order, one
// host-to-device copy per tensor (pieces of at most one slot for tensors
// larger than a slot), two stages with one item in each -- the host copy of
// tensor i+1 into the pinned ring overlaps the DMA of tensor i, and the DMAs
// run back to back on one copy stream, straight into the destinations. A
// slot is packed with consecutive pieces until full; it is refilled once the
// copy stream has finished reading it. A pinned blob is copied tensor by
// tensor without staging.
static int run_pertensor(ii_plan_t* p, const uint8_t* blob, const uint64_t* dst,
                         hipStream_t stream) {
    int rc = ensure_state(p);
    if (rc) return rc;
    rc = ensure_ring(p);
    if (rc) return rc;
    Runtime* r = p->rt;
    rc = check_dst(p, dst);
    if (rc) return rc;
    const bool pinned = pinned_span(p, blob);
    hipStream_t cs = r->lane_s[0];
    II_HIP(hipEventRecord(r->entry, stream));
    II_HIP(hipStreamWaitEvent(cs, r->entry, 0));
    if (pinned) {
        // straight from the pinned blob, tensor by tensor (rows by one 2-D copy)
        for (size_t i = 0; i < p->nbytes.size(); ++i) {
            const uint64_t n = p->nbytes[i];
            if (!n) continue;
            const uint8_t* src = blob + p->src_offset[i];
            const uint64_t rb = n / p->rows[i];
            if (p->rows[i] > 1)
                II_HIP(h2d_2d(reinterpret_cast<void*>(dst[i]), rb, src, p->row_stride[i], rb,
                              p->rows[i], cs));
            else
                II_HIP(h2d(reinterpret_cast<void*>(dst[i]), src, n, cs));
        }
    } else {
        // through the pinned slots (pertensor.h): slot 0 may still be read by
        // the previous load's copies
        if (r->copy_rec[0]) II_HIP(hipEventSynchronize(r->copy_done[0]));
        auto stage = [&](uint32_t slot, uint64_t at, size_t i, uint64_t src_rel,
                         uint64_t len) -> int {
            r->pool->copy(r->hslot[slot] + at, blob + p->src_offset[i] + src_rel, len);
            return II_OK;
        };
        auto copy = [&](uint32_t slot, uint64_t at, size_t i, uint64_t toff, uint64_t len) -> int {
            II_HIP(h2d(reinterpret_cast<void*>(dst[i] + toff), r->hslot[slot] + at, len, cs));
            return II_OK;
        };
        auto close = [&](uint32_t slot, uint32_t next) -> int {
            II_HIP(hipEventRecord(r->copy_done[slot], cs));
            r->copy_rec[slot] = 1;
            if (next < r->depth && r->copy_rec[next])
                II_HIP(hipEventSynchronize(r->copy_done[next]));
            return II_OK;
        };
        rc = pertensor_schedule(p->nbytes.data(), p->rows.data(), p->row_stride.data(),
                                p->nbytes.size(), p->chunk_bytes, r->depth, stage, copy, close);
        if (rc) return rc;
    }
    II_HIP(hipEventRecord(r->done, cs));
    II_HIP(hipStreamWaitEvent(stream, r->done, 0));
    return II_OK;
}

}  // namespace ii

using namespace ii;

extern "C" int ii_load_pertensor(ii_plan_t* p, const void* host_blob, uint64_t blob_bytes,
                                 void* const* dst_ptrs, hipStream_t stream) {
    if (!p) return fail(II_EINVAL, "ii_load_pertensor: plan is NULL");
    const size_t n = p->nbytes.size();
    if (n && !dst_ptrs) return fail(II_EINVAL, "ii_load_pertensor: dst_ptrs is NULL");
    if (p->num_chunks && !host_blob) return fail(II_EINVAL, "ii_load_pertensor: host_blob is NULL");
    if (blob_bytes < p->hi)
        return fail(II_ERANGE, "ii_load_pertensor: blob has %llu bytes, plan needs %llu",
                    (unsigned long long)blob_bytes, (unsigned long long)p->hi);
    if (p->num_chunks && is_device_ptr(host_blob))
        return fail(II_EINVAL, "ii_load_pertensor: host_blob is device memory");
    BusyGuard g(p);
    if (!g.ok) return fail(II_EBUSY, "ii_load_pertensor: plan in use");
    inject_arm();
    int rc = run_pertensor(p, static_cast<const uint8_t*>(host_blob),
                           reinterpret_cast<const uint64_t*>(dst_ptrs), stream);
    return rc ? drain(p, stream, rc) : II_OK;
}

extern "C" int ii_load(ii_plan_t* p, const void* host_blob, uint64_t blob_bytes,
                       void* const* dst_ptrs, hipStream_t stream) {
    if (!p) return fail(II_EINVAL, "ii_load: plan is NULL");
    const size_t n = p->nbytes.size();
    if (n && !dst_ptrs) return fail(II_EINVAL, "ii_load: dst_ptrs is NULL");
    if (p->num_chunks && !host_blob) return fail(II_EINVAL, "ii_load: host_blob is NULL");
    if (blob_bytes < p->hi)
        return fail(II_ERANGE, "ii_load: blob has %llu bytes, plan needs %llu",
                    (unsigned long long)blob_bytes, (unsigned long long)p->hi);
    if (p->num_chunks && is_device_ptr(host_blob))
        return fail(II_EINVAL, "ii_load: host_blob is device memory (use ii_load_device)");
    BusyGuard g(p);
    if (!g.ok) return fail(II_EBUSY, "ii_load: plan in use");
    inject_arm();
    Source src;
    src.blob = static_cast<const uint8_t*>(host_blob);
    int rc = run_ring(p, src, reinterpret_cast<const uint64_t*>(dst_ptrs), stream, nullptr);
    return rc ? drain(p, stream, rc) : II_OK;
}

extern "C" int ii_load_file(ii_plan_t* p, int fd, uint64_t file_bytes, void* const* dst_ptrs,
                            hipStream_t stream) {
    if (!p) return fail(II_EINVAL, "ii_load_file: plan is NULL");
    const size_t n = p->nbytes.size();
    if (n && !dst_ptrs) return fail(II_EINVAL, "ii_load_file: dst_ptrs is NULL");
    if (p->num_chunks && fd < 0) return fail(II_EINVAL, "ii_load_file: bad file descriptor");
    if (file_bytes < p->hi)
        return fail(II_ERANGE, "ii_load_file: file has %llu bytes, plan needs %llu",
                    (unsigned long long)file_bytes, (unsigned long long)p->hi);
    Source src;
    src.fd = fd;
    if (p->num_chunks) {
        const int fl = fcntl(fd, F_GETFL);
        if (fl < 0) return fail(II_EINVAL, "ii_load_file: fcntl: %s", strerror(errno));
        src.direct = (fl & O_DIRECT) != 0;
    }
    BusyGuard g(p);
    if (!g.ok) return fail(II_EBUSY, "ii_load_file: plan in use");
    inject_arm();
    int rc = run_ring(p, src, reinterpret_cast<const uint64_t*>(dst_ptrs), stream, nullptr);
    return rc ? drain(p, stream, rc) : II_OK;
}

extern "C" int ii_load_device(ii_plan_t* p, const void* dev_image, uint64_t image_bytes,
                              void* const* dst_ptrs, hipStream_t stream) {
    if (!p) return fail(II_EINVAL, "ii_load_device: plan is NULL");
    const size_t n = p->nbytes.size();
    if (n && !dst_ptrs) return fail(II_EINVAL, "ii_load_device: dst_ptrs is NULL");
    if (p->num_chunks && !dev_image) return fail(II_EINVAL, "ii_load_device: dev_image is NULL");
    if (image_bytes < p->hi)
        return fail(II_ERANGE, "ii_load_device: image has %llu bytes, plan needs %llu",
                    (unsigned long long)image_bytes, (unsigned long long)p->hi);
    BusyGuard g(p);
    if (!g.ok) return fail(II_EBUSY, "ii_load_device: plan in use");
    inject_arm();
    int rc = run_device(p, static_cast<const uint8_t*>(dev_image),
                        reinterpret_cast<const uint64_t*>(dst_ptrs), stream);
    return rc ? drain(p, stream, rc) : II_OK;
}

extern "C" int ii_load_device_noalloc(ii_plan_t* p, const void* dev_image, uint64_t image_bytes,
                                      void* const* dst_ptrs, hipStream_t stream) {
    if (!p) return fail(II_EINVAL, "ii_load_device_noalloc: plan is NULL");
    const ScratchLayout l = scratch_layout(p);
    if (l.end > kScratchBytes)
        return fail(II_ESCRATCH, "ii_load_device_noalloc: the plan's tables need %llu bytes, the "
                    "static workspace holds %llu", (unsigned long long)l.end,
                    (unsigned long long)kScratchBytes);
    const size_t n = p->nbytes.size();
    if (n && !dst_ptrs) return fail(II_EINVAL, "ii_load_device_noalloc: dst_ptrs is NULL");
    if (p->num_chunks && !dev_image)
        return fail(II_EINVAL, "ii_load_device_noalloc: dev_image is NULL");
    if (image_bytes < p->hi)
        return fail(II_ERANGE, "ii_load_device_noalloc: image has %llu bytes, plan needs %llu",
                    (unsigned long long)image_bytes, (unsigned long long)p->hi);
    BusyGuard g(p);
    if (!g.ok) return fail(II_EBUSY, "ii_load_device_noalloc: plan in use");
    inject_arm();
    int rc = run_device_noalloc(p, static_cast<const uint8_t*>(dev_image),
                                reinterpret_cast<const uint64_t*>(dst_ptrs), stream);
    return rc ? drain(p, stream, rc) : II_OK;
}

// Bytes of the old layout's tensor ranges that no new tensor covers, as
// device address ranges inside the arena, split into pieces of at most
// 1 MiB (one workgroup each).
static std::vector<RangeDev> scrub_ranges(const ii_plan_t* po, const ii_plan_t* pn, uint64_t arena) {
    std::vector<std::pair<uint64_t, uint64_t>> olds, news;
    for (size_t i = 0; i < po->nbytes.size(); ++i)
        if (po->nbytes[i]) olds.push_back({po->dst_offset[i], po->dst_offset[i] + po->nbytes[i]});
    for (size_t i = 0; i < pn->nbytes.size(); ++i)
        if (pn->nbytes[i]) news.push_back({pn->dst_offset[i], pn->dst_offset[i] + pn->nbytes[i]});
    // both layouts are in increasing, non-overlapping order by construction
    std::vector<RangeDev> out;
    const uint64_t piece = 1u << 20;
    size_t j = 0;
    for (auto [b, e] : olds) {
        uint64_t x = b;
        while (j < news.size() && news[j].second <= x) ++j;
        size_t jj = j;
        while (x < e) {
            uint64_t y = e;
            if (jj < news.size() && news[jj].first < e) y = std::max(x, news[jj].first);
            for (uint64_t c = x; c < y; c += piece)
                out.push_back(RangeDev{arena + c, arena + std::min(y, c + piece)});
            if (jj < news.size() && news[jj].first < e) {
                x = std::max(x, news[jj].second);
                ++jj;
            } else {
                x = e;
            }
        }
    }
    return out;
}

extern "C" int ii_switch(const ii_plan_t* po, ii_plan_t* pn, void* arena, uint64_t arena_bytes,
                         const void* host_blob_new, uint64_t blob_bytes, hipStream_t stream) {
    if (!po || !pn) return fail(II_EINVAL, "ii_switch: plan is NULL");
    if (!arena) return fail(II_EINVAL, "ii_switch: arena is NULL");
    if (arena_bytes < pn->arena_bytes || arena_bytes < po->arena_bytes)
        return fail(II_EARENA, "ii_switch: arena has %llu bytes, plans need %llu (new) / %llu (old)",
                    (unsigned long long)arena_bytes, (unsigned long long)pn->arena_bytes,
                    (unsigned long long)po->arena_bytes);
    const uint64_t a = reinterpret_cast<uint64_t>(arena);
    if (a & (pn->max_align - 1))
        return fail(II_EALIGN, "ii_switch: arena not aligned to %llu",
                    (unsigned long long)pn->max_align);
    // the scrub writes anywhere in the old layout, so the whole arena the
    // caller declares must be memory the device can write
    uint64_t arena_end;
    if (__builtin_add_overflow(a, arena_bytes, &arena_end))
        return fail(II_EOVERFLOW, "ii_switch: arena + arena_bytes overflows");
    if (arena_bytes && !accessible(a, arena_end))
        return fail(II_EINVAL, "ii_switch: the arena [%#llx, +%llu bytes) is not memory the "
                    "device can write: not inside one device allocation or pinned host memory",
                    (unsigned long long)a, (unsigned long long)arena_bytes);
    if (pn->num_chunks && !host_blob_new) return fail(II_EINVAL, "ii_switch: host blob is NULL");
    if (blob_bytes < pn->hi)
        return fail(II_ERANGE, "ii_switch: blob has %llu bytes, plan needs %llu",
                    (unsigned long long)blob_bytes, (unsigned long long)pn->hi);
    if (pn->num_chunks && is_device_ptr(host_blob_new))
        return fail(II_EINVAL, "ii_switch: host blob is device memory");
    BusyGuard g(pn);
    if (!g.ok) return fail(II_EBUSY, "ii_switch: plan in use");
    inject_arm();
    std::vector<uint64_t> dst(pn->nbytes.size());
    for (size_t i = 0; i < dst.size(); ++i) dst[i] = a + pn->dst_offset[i];
    std::vector<RangeDev> scrub = scrub_ranges(po, pn, a);
    Source src;
    src.blob = static_cast<const uint8_t*>(host_blob_new);
    int rc = run_ring(pn, src, dst.data(), stream, &scrub);
    return rc ? drain(pn, stream, rc) : II_OK;
}

extern "C" int ii_plan_set_ring(ii_plan_t* p, uint32_t depth, uint32_t host_threads,
                                uint32_t copy_streams) {
    if (!p) return fail(II_EINVAL, "ii_plan_set_ring: plan is NULL");
    if (depth < 1 || depth > 8 || host_threads < 1 || host_threads > 64 || copy_streams < 1 ||
        copy_streams > kMaxLanes || copy_streams > depth)
        return fail(II_EINVAL, "ii_plan_set_ring: depth must be 1..8, host_threads 1..64, "
                               "copy_streams 1..min(4, depth)");
    if (p->rt && p->rt->depth) return fail(II_EBUSY, "ii_plan_set_ring: ring already allocated");
    p->ring_depth = depth;
    p->host_threads = host_threads;
    p->copy_streams = copy_streams;
    return II_OK;
}

extern "C" int ii_plan_set_trace(ii_plan_t* p, int on) {
    if (!p) return fail(II_EINVAL, "ii_plan_set_trace: plan is NULL");
    p->trace = on != 0;
    return II_OK;
}

extern "C" int ii_plan_trace(ii_plan_t* p, float* copy_start, float* copy_end,
                             float* scatter_start, float* scatter_end) {
    if (!p) return fail(II_EINVAL, "ii_plan_trace: plan is NULL");
    Runtime* r = p->rt;
    if (!r || !r->tr_chunks)
        return fail(II_EINVAL, "ii_plan_trace: no traced ring load on record");
    BusyGuard g(p);
    if (!g.ok) return fail(II_EBUSY, "ii_plan_trace: plan in use");
    const size_t L = r->tr_chunks;
    II_HIP(hipEventSynchronize(r->tr_se[L - 1]));
    for (float* out : {copy_start, copy_end, scatter_start, scatter_end})
        if (out)
            for (size_t k = 0; k < p->num_chunks; ++k) out[k] = std::nanf("");
    for (size_t j = 0; j < L; ++j) {
        const uint32_t k = r->tr_id[j];
        const struct {
            float* out;
            hipEvent_t e;
        } items[4] = {{copy_start, r->tr_cs[j]}, {copy_end, r->tr_ce[j]},
                      {scatter_start, r->tr_ss[j]}, {scatter_end, r->tr_se[j]}};
        for (const auto& it : items) {
            if (!it.out) continue;
            II_HIP(hipEventSynchronize(it.e));
            II_HIP(hipEventElapsedTime(&it.out[k], r->tr_t0, it.e));
        }
    }
    return II_OK;
}

extern "C" int ii_check_dst(const ii_plan_t* p, void* const* dst_ptrs) {
    if (!p) return fail(II_EINVAL, "ii_check_dst: plan is NULL");
    if (p->nbytes.size() && !dst_ptrs) return fail(II_EINVAL, "ii_check_dst: dst_ptrs is NULL");
    return check_dst(p, reinterpret_cast<const uint64_t*>(dst_ptrs));
}

extern "C" int ii_plan_prepare(ii_plan_t* p) {
    if (!p) return fail(II_EINVAL, "ii_plan_prepare: plan is NULL");
    BusyGuard g(p);
    if (!g.ok) return fail(II_EBUSY, "ii_plan_prepare: plan in use");
    inject_arm();
    int rc = ensure_state(p);
    if (rc) return rc;
    rc = ensure_ring_tables(p);
    if (rc) return rc;
    return ensure_ring(p);
}

extern "C" int ii_plan_release(ii_plan_t* p) {
    if (!p) return fail(II_EINVAL, "ii_plan_release: plan is NULL");
    BusyGuard g(p);
    if (!g.ok) return fail(II_EBUSY, "ii_plan_release: plan in use");
    runtime_destroy(p);
    return II_OK;
}

extern "C" int ii_host_alloc(uint64_t bytes, void** out) {
    if (!out) return fail(II_EINVAL, "ii_host_alloc: out is NULL");
    *out = nullptr;
    if (!bytes) return II_OK;
    II_HIP(hipHostMalloc(out, bytes, 0));
    return II_OK;
}

extern "C" int ii_host_free(void* ptr) {
    if (!ptr) return II_OK;
    II_HIP(hipHostFree(ptr));
    return II_OK;
}
