/*
 * ii.h -- merged tensor loading on AMD Instinct MI355X (gfx950).
 *
 * C-ABI of libii.so. The library implements the refined tensor
 * materialisation of InstantInfer (arXiv 2607.18957, Sec. 4.2): instead of
 * one small host-to-device copy per tensor, the bytes of a weight blob are cut
 * into a few large equal chunks, each chunk is streamed host -> HBM in bulk
 * through a pinned staging ring, and a device kernel scatters the chunk into
 * every tensor it holds while the next chunk is still in flight.
 *
 * Conventions for every entry point:
 *   - Return value: II_OK (0) or one of the II_E* codes below. On error a
 *     thread-local description is available from ii_last_error().
 *   - Pointers are plain host or device addresses; sizes are bytes.
 *   - Nothing here allocates on behalf of the caller except ii_host_alloc and
 *     the plan's own staging buffers (see ii_load).
 *   - A plan is not thread-safe: two calls that use the same plan at the same
 *     time from different host threads get II_EBUSY for the later one.
 */
#ifndef II_H
#define II_H

#include <stddef.h>
#include <stdint.h>

/* The HIP stream handle, declared exactly as the HIP runtime declares it, so
 * this header needs no ROCm include path; repeating the typedef alongside
 * <hip/hip_runtime_api.h> is harmless. */
typedef struct ihipStream_t* hipStream_t;

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ------------------------------------------------------ */
enum {
    II_OK = 0,
    II_EINVAL = 1,    /* NULL argument, bad chunk size, bad dtype/shape/alignment,
                         memory the device cannot reach */
    II_EOVERFLOW = 2, /* a byte size or offset does not fit in 64 bits */
    II_EOVERLAP = 3,  /* source ranges overlap, or destination ranges overlap */
    II_EALIGN = 4,    /* a destination pointer is not aligned to its dst_align */
    II_ENOMEM = 5,    /* host or device allocation failed */
    II_EARENA = 6,    /* the arena is smaller than the new plan's arena_bytes */
    II_EBUSY = 7,     /* the plan is in use by another call */
    II_EHIP = 8,      /* any other HIP runtime error (detail in ii_last_error) */
    II_ERANGE = 9,    /* the blob, image or file is shorter than the plan's span end */
    II_EIO = 10,      /* reading the model file failed (detail in ii_last_error) */
    II_ESCRATCH = 11  /* the plan's tables exceed the static workspace of
                         ii_load_device_noalloc */
};

/* ---- element types (storage width in brackets) ---------------------------- */
enum {
    II_U8 = 1,       /* [1] */
    II_I8 = 2,       /* [1] */
    II_FP8_E4M3 = 3, /* [1] */
    II_FP8_E5M2 = 4, /* [1] */
    II_BF16 = 5,     /* [2] */
    II_F16 = 6,      /* [2] */
    II_F32 = 7,      /* [4] */
    II_I32 = 8,      /* [4] */
    II_F64 = 9,      /* [8] */
    II_I64 = 10      /* [8] */
};

/*
 * One row of the tensor table: a tensor's logical description and where its
 * bytes sit in the blob (the model file image in host memory; in the paper,
 * the checkpoint read from storage or tmpfs, Sec. 5).
 *   name        optional, may be NULL; copied by ii_plan.
 *   dtype       one of the II_* element types above.
 *   ndim        number of dimensions (0 = scalar).
 *   shape       ndim non-negative extents; copied by ii_plan. nbytes =
 *               product(shape) x width(dtype). Zero-size tensors are allowed.
 *   src_offset  byte offset of the tensor's first byte in the blob.
 *   dst_align   required alignment (power of two) of the tensor's
 *               destination address.
 *   src_row_stride
 *               0: the tensor's bytes are contiguous in the blob. Otherwise
 *               the tensor is shape[0] rows of nbytes / shape[0] bytes each,
 *               row q starting at blob byte src_offset + q * src_row_stride
 *               (a column block of a larger row-major matrix, as a
 *               tensor-parallel rank holds its shard of a row-parallel weight
 *               in an unsharded model file; Sec. 2.2, Sec. 6.1). The
 *               destination is always contiguous: row q lands at tensor byte
 *               q * (nbytes / shape[0]). Requires ndim >= 1 and, when
 *               shape[0] > 1, src_row_stride >= the row's bytes; ignored for
 *               zero-size tensors. Rows of different tensors may interleave
 *               but no blob byte may belong to two rows.
 */
typedef struct ii_tensor_desc {
    const char* name;
    int32_t dtype;
    int32_t ndim;
    const int64_t* shape;
    uint64_t src_offset;
    uint64_t dst_align;
    uint64_t src_row_stride;
} ii_tensor_desc;

typedef struct ii_plan_s ii_plan_t; /* opaque */

/*
 * ii_plan -- precompute the chunk <-> tensor association (Sec. 4.2, "Refined
 * CFA Model": the file is divided into equal-length chunks, the last one
 * possibly partial, and the tensor.chunks / chunk.tensors maps are computed in
 * advance).
 *
 * Chunks are windows of chunk_bytes over the span [lo, hi) of the table's
 * source bytes (lo = smallest source offset, hi = largest source end over
 * non-empty tensors, or over their rows for tensors given with a row
 * stride); chunk k covers [lo + k*chunk_bytes, min(lo + (k+1)*chunk_bytes,
 * hi)). A segment is one tensor's piece of one chunk (for a tensor given as
 * rows, one row's piece of one chunk), ordered by offset in the chunk.
 * The ring loads skip chunks that hold no segment, and move of each other
 * chunk only its segment bytes (gathered on the host, or copied from a
 * pinned blob row group by row group) or the range from its first segment's
 * start to its last segment's end (see ii_plan_copy_bytes).
 * The scatter kernel's tiles take 4096 segment bytes each ($II_TILE_BYTES,
 * read by ii_plan, overrides it: 1024..65536, rounded down to a multiple of
 * 16).
 * Destination layout (used by ii_switch and by callers carving an arena): in
 * table order, tensor i starts at the smallest multiple of dst_align[i] at or
 * after the end of tensor i-1; arena_bytes is the end rounded up to the
 * largest alignment.
 *
 *   table        n rows; read only during the call (names and shapes copied).
 *   n            number of rows; 0 is valid (a plan with no chunks).
 *   chunk_bytes  chunk size: a multiple of 16, 16 <= chunk_bytes < 2^32.
 *   out          receives the plan; release with ii_plan_free.
 * Host only: touches no device. Errors: II_EINVAL (NULL out, NULL table with
 * n > 0, bad chunk_bytes, unknown dtype, negative ndim or extent, dst_align
 * not a power of two, a row stride on a scalar or shorter than its row, more
 * than 2^31 rows in all), II_EOVERFLOW (a size or a source end, including a
 * last row's end, does not fit in 64 bits), II_EOVERLAP (two non-empty
 * source ranges or rows share a byte), II_ENOMEM.
 */
int ii_plan(const ii_tensor_desc* table, size_t n, uint64_t chunk_bytes, ii_plan_t** out);

/* Release a plan and everything it owns (staging rings, device tables).
 * Waits for the plan's outstanding device work first. NULL is a no-op. */
void ii_plan_free(ii_plan_t* plan);

/*
 * ii_load -- materialise every tensor of the plan from a host blob into
 * device memory (Sec. 4.2). For each chunk that holds a segment, in order:
 * bring its bytes into a pinned host slot (its used range, or only its
 * segments' bytes, packed, when it has gaps between segments), copy it to a
 * device slot with one hipMemcpyAsync, then scatter it into its tensors
 * with the device kernel. A pinned blob's chunk skips the host slot: it is
 * copied straight from the blob -- its used range in one copy, or, when it
 * has gaps, its run groups in one 1-D or 2-D copy each (see
 * ii_plan_copy_bytes; a chunk of many groups that is mostly gaps is still
 * gathered through the host slot).
 * Chunks holding no segment are not touched. Chunk k's copy and scatter
 * run on lane k mod lanes (see ii_plan_set_ring), so with two or more lanes
 * chunk k+1's copy overlaps chunk k's scatter. A slot is
 * reused only after the scatter that read it has finished (Sec. 4.2:
 * (C_i,InMem)->(C_i+1,InDisk), (C_i,InGPU)->(C_i+1,InMem),
 * (C_i,InGPU)->(T_j,Alloc), (T_j,Loaded)->(C_i,InGPU)).
 *
 *   plan        from ii_plan. On first use it allocates, on the current
 *               device, a ring of `depth` pinned host slots and `depth`
 *               device slots of chunk_bytes each (default depth 3, see
 *               ii_plan_set_ring) plus the plan's device tables; they are
 *               kept for later loads until ii_plan_release / ii_plan_free.
 *   host_blob   host address of blob byte 0. Pageable or pinned. Pageable
 *               blobs are read only during the call; a pinned blob
 *               (hipHostMalloc / ii_host_alloc) is read by DMA after the call
 *               returns and must stay valid and unchanged until `stream`
 *               reaches the point after this call. A blob counts as pinned
 *               when the first and the last byte of the span [lo, hi) are
 *               pinned; otherwise it is handled as pageable.
 *   blob_bytes  size of the blob; must be >= the plan's span end hi.
 *   dst_ptrs    n device addresses, one per table row (NULL allowed only for
 *               zero-size tensors); dst_ptrs[i] must be a multiple of
 *               dst_align[i]; the ranges [dst_ptrs[i], +nbytes[i]) must not
 *               overlap, and each must lie inside one device allocation or
 *               in pinned host memory (checked, II_EINVAL; see
 *               ii_check_dst). Read during the call only; the memory they
 *               point to must stay allocated until `stream` passes this
 *               call.
 *   stream      HIP stream (0 = null stream). Writes into the destinations
 *               start only after all work already enqueued on `stream`, and
 *               complete before any work enqueued on `stream` afterwards.
 * Only the tensors' bytes are written: destination padding and every other
 * byte are left untouched. Returns once all work is enqueued (for a
 * pageable blob also after its bytes have been staged). Errors: II_EINVAL,
 * II_EALIGN, II_EOVERLAP, II_ERANGE, II_ENOMEM, II_EBUSY, II_EHIP. After an
 * error nothing remains enqueued that writes caller memory and the plan stays
 * usable.
 */
int ii_load(ii_plan_t* plan, const void* host_blob, uint64_t blob_bytes, void* const* dst_ptrs,
            hipStream_t stream);

/*
 * ii_load_file -- the same materialisation with the blob read from a file
 * (the model file on storage or on tmpfs; Sec. 4.2 InDisk -> InMem, Sec. 5):
 * the host threads read each chunk's bytes (only its segments' bytes when it
 * has gaps: each thread's runs in batched preadv calls, run bytes straight
 * into place, gaps under 256 KiB into a scratch buffer) into a pinned slot,
 * then the copy and scatter steps run as in ii_load. If fd was opened
 * with O_DIRECT, every read starts and ends on a 4096-byte boundary and
 * bypasses the page cache; those reads land in a page-aligned host buffer
 * (device-pinned pages cannot be targets of direct I/O), read ahead by
 * several threads, from which the host threads copy (or gather) the chunk
 * into the pinned slot.
 *   fd          open for reading; file byte x is blob byte x. Read during the
 *               call only; the call returns once every chunk has been read.
 *   file_bytes  size of the file; must be >= the plan's span end hi.
 *   dst_ptrs, stream   as for ii_load.
 * Errors: as ii_load, plus II_EIO when a read fails or the file ends early.
 */
int ii_load_file(ii_plan_t* plan, int fd, uint64_t file_bytes, void* const* dst_ptrs,
                 hipStream_t stream);

/*
 * ii_load_device -- the same materialisation from a blob image that is
 * already resident in device memory (for example a checkpoint image parked in
 * HBM): no staging and no host-to-device copy; every segment of every chunk
 * is copied straight from the image into its tensor by one launch on
 * `stream` (the device half of Sec. 4.2, with all chunks resident at once).
 * The launch is cut by destination: each workgroup writes one window of
 * tile_bytes of the plan's destination layout (see ii_plan_layout_tiles).
 *
 *   dev_image    device address of blob byte 0 (any alignment); the span
 *                [dev_image + lo, + hi) must lie inside one device allocation
 *                or in pinned host memory (checked, II_EINVAL). From pinned
 *                host memory the kernel reads the blob over the host link
 *                itself: no ring and no copy engine, one launch -- the
 *                lowest latency for small loads.
 *   image_bytes  size of the image; must be >= the plan's span end hi.
 *   dst_ptrs     as for ii_load; must not overlap [dev_image, +hi).
 *   stream       the kernel runs on this stream, after the work already on
 *                it. The caller keeps the image and destinations alive
 *                until the stream passes this call.
 * Errors: as ii_load.
 */
int ii_load_device(ii_plan_t* plan, const void* dev_image, uint64_t image_bytes,
                   void* const* dst_ptrs, hipStream_t stream);

/*
 * ii_load_device_noalloc -- ii_load_device for callers that cannot allocate
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc): the same result, arguments, ordering and errors, but
 * the call allocates nothing -- no device or pinned host memory, no events,
 * streams or plan state. The kernel's tables (a 32-byte row per segment, an
 * 8-byte segment range per layout tile, and when some window of the layout
 * holds only padding a 4-byte window index per tile) are uploaded on every
 * call, on `stream`, into a static device workspace of 64 MiB that the
 * library holds on each GPU it runs on until the process ends; a plan whose
 * tables need more returns II_ESCRATCH before anything is checked or
 * enqueued (the Llama-8B-shaped table needs 31 MB, the 100,000-tensor one
 * 5.1 MB). Calls
 * on one GPU share that workspace: two calls ordered on one stream are
 * safe, calls that overlap on different streams of one GPU race (the later
 * upload may overwrite tables an earlier kernel still reads) and must be
 * ordered by the caller.
 * Errors: as ii_load_device, plus II_ESCRATCH.
 */
int ii_load_device_noalloc(ii_plan_t* plan, const void* dev_image, uint64_t image_bytes,
                           void* const* dst_ptrs, hipStream_t stream);

/*
 * ii_load_pertensor -- the same result as ii_load by the naive per-tensor
 * pipeline of Sec. 4.2 ("Naive CFA Model"): one host-to-device copy per
 * tensor (a tensor larger than chunk_bytes is copied in chunk_bytes pieces;
 * a tensor given as rows is gathered row by row into the staging slot, or
 * from a pinned blob copied with one 2-D copy), in table order, straight
 * into its destination; the host staging of tensor
 * i+1 into the plan's pinned ring overlaps the copy of tensor i, and the
 * copies run one after another on one copy stream ((T_i,InMem) ->
 * (T_i+1,InDisk) and (T_i,InGPU) -> (T_i+1,InMem)). No scatter kernel runs.
 * It exists to measure what merging saves; arguments, ordering, ownership
 * and errors are exactly those of ii_load.
 */
int ii_load_pertensor(ii_plan_t* plan, const void* host_blob, uint64_t blob_bytes,
                      void* const* dst_ptrs, hipStream_t stream);

/*
 * ii_switch -- reuse a device arena that holds plan_old's tensors (at
 * plan_old's layout offsets) for plan_new's tensors (at plan_new's offsets),
 * following the model-switch dependency (Sec. 4.3): the new model's
 * preparation that does not need the arena (staging and host-to-device
 * copies into the ring) starts at once, while the first write into the arena
 * waits for all work enqueued on `stream` before this call, i.e. for the old
 * model to have finished with its memory, (M1,GMemFreed)->(M2,EnvReady).
 * Afterwards every byte of a new tensor holds the new blob's bytes, every
 * byte that belonged to an old tensor and to no new tensor is zero, and all
 * other arena bytes are untouched.
 *
 *   plan_old     layout of what the arena holds now (only its layout is used).
 *   plan_new     the table to load; its ring and tables are used as in ii_load.
 *   arena        device address, aligned to plan_new's largest dst_align.
 *   arena_bytes  must be >= both plans' arena_bytes, else II_EARENA; the
 *                whole range [arena, arena + arena_bytes) must lie inside
 *                one device allocation (or in pinned host memory), else
 *                II_EINVAL, since the scrub may write anywhere in the old
 *                layout.
 *   host_blob_new, blob_bytes, stream   as for ii_load.
 * Errors: as ii_load, plus II_EARENA, and II_EOVERFLOW when arena +
 * arena_bytes does not fit in 64 bits; all checks run before anything is
 * enqueued.
 */
int ii_switch(const ii_plan_t* plan_old, ii_plan_t* plan_new, void* arena, uint64_t arena_bytes,
              const void* host_blob_new, uint64_t blob_bytes, hipStream_t stream);

/*
 * Ring configuration, before the plan's first load or after
 * ii_plan_release. depth = number of chunk slots in flight (1..8; default 3
 * or $II_RING_DEPTH); host_threads = threads that read, copy or gather
 * chunk bytes into the pinned slots (pageable blobs, files, gathered chunks;
 * 1..64; default min(8, cores) or $II_HOST_THREADS);
 * copy_streams = lanes, the streams the chunks alternate between (1..min(4,
 * depth); default min(depth, 3) or $II_COPY_STREAMS): chunk k's host-to-device copy and
 * then its scatter run on lane k mod copy_streams. With 1, copies and
 * scatters alternate on one stream in chunk order; with more, the copy of
 * one chunk overlaps the scatter of another, and a slot whose next chunk
 * runs on another lane is handed over by an event. Each lane's first copy
 * of a load may run before the work the caller enqueued ahead of it.
 * Errors: II_EINVAL (out of range), II_EBUSY (ring already allocated).
 */
int ii_plan_set_ring(ii_plan_t* plan, uint32_t depth, uint32_t host_threads,
                     uint32_t copy_streams);

/*
 * ii_check_dst -- the destination checks every load runs, without loading:
 * each non-empty tensor's pointer is non-NULL and aligned to its dst_align,
 * the ranges [dst_ptrs[i], +nbytes[i]) are pairwise disjoint, and each lies
 * inside one device allocation (or in pinned host memory). Touches no
 * device memory. Errors: II_EINVAL (NULL arguments, a pointer the device
 * cannot write, with the tensor named in ii_last_error), II_EALIGN,
 * II_EOVERLAP, II_EOVERFLOW.
 */
int ii_check_dst(const ii_plan_t* plan, void* const* dst_ptrs);

/*
 * ii_plan_prepare -- allocate, on the current device, what the plan's loads
 * would otherwise allocate on first use: the staging ring (pinned host slots,
 * touched page by page so the first load does not fault them in; device
 * slots; streams; host copy threads) and the ring's device tables (the
 * resident-image kernel's tables are allocated by the first ii_load_device
 * that needs them). Optional:
 * a cold-starting process can call it while other initialisation runs, so
 * the first load starts moving bytes at once (Sec. 4.2 overlaps independent
 * steps of the cold start). Idempotent. Errors: II_EINVAL (NULL plan, or a
 * plan first used on another device), II_EBUSY, II_ENOMEM, II_EHIP.
 */
int ii_plan_prepare(ii_plan_t* plan);

/*
 * Pipeline timeline. With tracing on (ii_plan_set_trace(plan, 1) or
 * $II_TRACE=1), every later ii_load / ii_switch on the plan records four
 * timing events per chunk k: before and after its host-to-device copy and
 * before and after its scatter (on its lane). ii_plan_trace waits for the
 * last traced load to finish and writes, for each chunk, the times in
 * milliseconds since the point where that load's destination writes may
 * begin (after the work the caller enqueued ahead of it; a copy that ran
 * before that point has a negative time) into arrays of num_chunks entries
 * (NULL skips one); chunks that hold no segment are not moved and get NaN.
 * The dependency edges can be read off them: copy_end[k] <= scatter_start[k],
 * and scatter_end of the i-th moved chunk <= copy_start of the (i +
 * depth)-th. Errors: II_EINVAL (tracing off or no traced load), II_EBUSY,
 * II_EHIP.
 */
int ii_plan_set_trace(ii_plan_t* plan, int on);
int ii_plan_trace(ii_plan_t* plan, float* copy_start, float* copy_end, float* scatter_start,
                  float* scatter_end);

/* Free the plan's staging ring and device tables after waiting for its
 * outstanding work (the paper frees its I/O buffers as soon as loading
 * completes, Sec. 6.6). The plan stays valid; the next load reallocates. */
int ii_plan_release(ii_plan_t* plan);

/* ---- plan inspection (host only) ----------------------------------------- */
size_t ii_plan_num_tensors(const ii_plan_t* plan);
size_t ii_plan_num_chunks(const ii_plan_t* plan);
size_t ii_plan_num_segments(const ii_plan_t* plan);
uint64_t ii_plan_chunk_bytes(const ii_plan_t* plan);
uint64_t ii_plan_payload_bytes(const ii_plan_t* plan); /* sum of nbytes */
uint64_t ii_plan_arena_bytes(const ii_plan_t* plan);
/* bytes one ii_load from a pinned blob moves from host to device. A table
 * whose tensors tile their span: per chunk, its used range -- first
 * segment's start to last segment's end, rounded out to 256-byte boundaries
 * inside the chunk -- copied in place (hi - lo in all). A table with gaps
 * between segments: per chunk that holds segments, only its segment bytes
 * when its runs (segments adjacent in the file, merged) form at most 2
 * groups of one run length and one spacing ($II_PINNED_GROUPS_MAX, 0..64)
 * -- each group is one 1-D or 2-D copy straight from the blob (the rows of
 * a column block) -- or when more than a quarter of its used range is gaps
 * (it is then gathered on the host through the staging slot); otherwise its
 * used range in place. Loads from a pageable blob or a file gather every
 * chunk with gaps and move payload_bytes. */
uint64_t ii_plan_copy_bytes(const ii_plan_t* plan);
/* Packed staging layout (loads from a pageable blob or a file gather only
 * the segments' bytes of a chunk into its pinned slot, back to back in
 * segment order; a pinned blob's group copies land in the same layout): per
 * segment its offset in the slot (num_segments), per chunk the bytes staged
 * (num_chunks). For a table whose tensors tile their
 * span this equals the chunk layout. NULL skips a field. Errors: II_EINVAL
 * (NULL plan). */
int ii_plan_packing(const ii_plan_t* plan, uint32_t* seg_off, uint64_t* chunk_len);
/* span [lo, hi) of source bytes; both 0 when every tensor is empty */
void ii_plan_span(const ii_plan_t* plan, uint64_t* lo, uint64_t* hi);
/* per tensor (arrays of num_tensors; NULL skips a field) */
int ii_plan_tensors(const ii_plan_t* plan, uint64_t* nbytes, uint64_t* dst_offset);
/* per chunk (arrays of num_chunks; seg_begin has num_chunks + 1 entries: the
 * segments of chunk k are [seg_begin[k], seg_begin[k+1])) */
int ii_plan_chunks(const ii_plan_t* plan, uint64_t* src_begin, uint64_t* len,
                   uint64_t* seg_begin);
/* per segment, ordered by chunk then by offset in the chunk (arrays of
 * num_segments) */
int ii_plan_segments(const ii_plan_t* plan, uint32_t* chunk, uint32_t* chunk_off,
                     uint32_t* tensor, uint64_t* tensor_off, uint32_t* len);
/* the ring's work split (the scatter of one chunk in its staging slot, or
 * read in place), one workgroup per tile, tiles in chunk order:
 * tile g takes tile_bytes of its chunk's segment bytes (counted in segment
 * order, gaps between segments skipped; the chunk's last tile takes the
 * rest) and meets exactly the segments [first[g], last[g]). In a packed
 * staging slot those bytes are slot offsets [m * tile_bytes, ...), m = g's
 * index within its chunk; in the chunk itself they are the chunk offsets
 * [w0[g], w1[g]). A chunk without segments has no tiles. Arrays of
 * *num_tiles entries; pass NULL arrays to read only the sizes. */
int ii_plan_tiles(const ii_plan_t* plan, uint32_t* tile_bytes, uint64_t* num_tiles,
                  uint32_t* chunk, uint32_t* first, uint32_t* last, uint32_t* w0, uint32_t* w1);
/* the resident-image kernel's work split (ii_load_device), one workgroup per
 * tile, cut by destination: seg_order (num_segments entries) lists the
 * segments by layout position -- dst_offset of its tensor plus its tensor
 * offset -- and tile g takes the layout positions [window[g] * tile_bytes,
 * (window[g] + 1) * tile_bytes) and meets exactly the segments
 * seg_order[first[g]] .. seg_order[last[g] - 1]. Windows that hold only
 * padding have no tile. A unit of work (one segment's piece of one 16-byte
 * destination block) belongs to the tile whose window holds the layout
 * position of its first byte, so each destination byte is written by
 * exactly one workgroup whatever addresses the load passes. Arrays of
 * *num_tiles entries (seg_order: num_segments); NULL skips a field.
 * Errors: II_EINVAL (NULL plan). */
int ii_plan_layout_tiles(const ii_plan_t* plan, uint64_t* num_tiles, uint32_t* seg_order,
                         uint32_t* first, uint32_t* last, uint32_t* window);
/* which of its two variants the resident-image kernel runs for this plan: 1
 * for the variant for tables of many small tensors (tiles that one segment
 * meets take a path without LDS staging, and every tile issues all its
 * loads before using any), chosen when at least II_LAYOUT_MIXED_PCT percent
 * (default 5; 0 = always, 101 = never) of the tiles meet three or more
 * segments, or when at least 3% meet two or more and most payload bytes
 * are phase-shifted (blob offset and layout position differ mod 16); 0 for
 * the other (fewer loads in flight, faster on tables of large tensors).
 * Both write the same bytes. 0 for a NULL plan. */
int ii_plan_layout_mixed(const ii_plan_t* plan);
/* name of row i as given to ii_plan ("" if none); valid while the plan lives */
const char* ii_plan_tensor_name(const ii_plan_t* plan, size_t i);

/* ---- pinned host memory for blobs ---------------------------------------- */
/* Page-locked, device-accessible host allocation (hipHostMalloc) of exactly
 * `bytes`; a blob placed here is copied by DMA without staging. */
int ii_host_alloc(uint64_t bytes, void** out);
int ii_host_free(void* ptr);

/* ---- errors ------------------------------------------------------------- */
const char* ii_strerror(int status);
/* Detail of the last error raised on the calling thread ("" if none). */
const char* ii_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* II_H */
