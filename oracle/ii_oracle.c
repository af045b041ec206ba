/*
 * Oracle for merged tensor loading -- TEST INFRASTRUCTURE ONLY.
 *
 * Only the tests, the package smoke check and the benchmark's CPU-baseline
 * leg may load this library. The product path (the C-ABI library and its
 * binding) never calls it and shares no code with it.
 *
 * What it computes, and where the paper defines it
 * (InstantInfer, arXiv 2607.18957):
 *
 *   - Loader result. The refactored (DAG CFA) loader must end in the same
 *     final state as the original sequential (Chain CFA) program (Sec. 3.3,
 *     Theorem 2; proof and Chain-CFA construction in Sec. 8). The sequential
 *     program materialises tensors one by one, copying each from the model
 *     file into its own buffer (Sec. 4.2, first paragraph). So the expected
 *     result is tensor i's bytes = blob[src_i, src_i + nbytes_i).
 *     -> orc_load_into, orc_load_alloc, orc_arena.
 *
 *   - Chunks and their tensor associations. The model file is cut into
 *     chunks of equal length, the last one possibly partial, and a tensor is
 *     associated with every chunk its content falls in; one tensor may span
 *     several chunks and one chunk may hold several tensors (Sec. 4.2,
 *     "Refined CFA Model"). -> orc_plan, by brute-force intersection of every
 *     chunk window with every tensor's source range.
 *
 *   - Model switch. The new model may use GPU memory only after the old one
 *     has released it, (M1, GMemFreed) -> (M2, EnvReady) (Sec. 4.3). The byte
 *     content after reusing an arena is not specified by the paper; this
 *     oracle takes the reading that old-tensor bytes not covered by a new
 *     tensor are zeroed, new-tensor bytes hold the new model's bytes and all
 *     other bytes are untouched. -> orc_switch.
 *
 *   - Tensor-parallel shards. A rank's shard of a weight sharded along its
 *     inner dimension is not contiguous in the model file: each of its
 *     shape[0] rows is a run of row bytes at a fixed stride (the paper notes
 *     that tensor parallelism fragments transfers, Sec. 2.2). The *_rows
 *     functions below take, per tensor, a row count and a source stride; a
 *     contiguous tensor is one row. The result is tensor i's rows, in order,
 *     back to back. -> orc_rows, orc_check_rows, orc_span_rows,
 *     orc_plan_rows, orc_load_rows_into, orc_arena_rows.
 *
 * Readings where the paper is silent (also listed in the design notes):
 *   R1 chunk windows start at lo = min source offset over non-empty tensors
 *      and end at hi = max source end; bytes outside [lo, hi) are never read;
 *   R4 destination layout is table order, each tensor's offset the smallest
 *      multiple of its dst_align at or after the previous tensor's end; the
 *      arena size is the end rounded up to the largest alignment;
 *   R8 overlapping source ranges are rejected;
 *   R9 zero-size tensors are valid, get an offset and touch no chunk.
 *
 * Everything is plain and sequential on purpose: no blocking, fusion or
 * reordering beyond the definitions above.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum {
    ORC_OK = 0,
    ORC_EINVAL = 1,
    ORC_EOVERFLOW = 2,
    ORC_EOVERLAP = 3,
    ORC_ERANGE = 4, /* a source range lies outside the given blob */
};

/* Element width in bytes for each type code of the table format:
 * u8 i8 fp8_e4m3 fp8_e5m2 -> 1; bf16 f16 -> 2; f32 i32 -> 4; f64 i64 -> 8. */
int orc_esize(int32_t dtype)
{
    switch (dtype) {
    case 1: case 2: case 3: case 4: return 1;
    case 5: case 6: return 2;
    case 7: case 8: return 4;
    case 9: case 10: return 8;
    default: return 0;
    }
}

/* nbytes = (product of dims) x element width, with overflow detection. */
int orc_nbytes(int32_t dtype, int32_t ndim, const int64_t* shape, uint64_t* out)
{
    int es = orc_esize(dtype);
    if (es == 0 || ndim < 0 || (ndim > 0 && !shape))
        return ORC_EINVAL;
    for (int32_t d = 0; d < ndim; ++d)
        if (shape[d] < 0)
            return ORC_EINVAL;
    uint64_t numel = 1;
    int zero = 0;
    for (int32_t d = 0; d < ndim; ++d) {
        uint64_t x = (uint64_t)shape[d];
        if (x == 0)
            zero = 1;
        if (!zero) {
            if (numel > UINT64_MAX / x)
                return ORC_EOVERFLOW;
            numel *= x;
        }
    }
    if (zero) {
        *out = 0;
        return ORC_OK;
    }
    if (numel > UINT64_MAX / (uint64_t)es)
        return ORC_EOVERFLOW;
    *out = numel * (uint64_t)es;
    return ORC_OK;
}

/* Per-tensor byte sizes for a columnar table. shape_start[i] indexes the
 * first of tensor i's ndim[i] dimensions in shape_flat. */
int orc_sizes(size_t n, const int32_t* dtype, const int32_t* ndim, const int64_t* shape_flat,
              const int64_t* shape_start, uint64_t* nbytes)
{
    for (size_t i = 0; i < n; ++i) {
        int rc = orc_nbytes(dtype[i], ndim[i], shape_flat ? shape_flat + shape_start[i] : NULL,
                            &nbytes[i]);
        if (rc)
            return rc;
    }
    return ORC_OK;
}

typedef struct {
    uint64_t begin, end;
} orc_range;

static int cmp_range(const void* a, const void* b)
{
    const orc_range* x = (const orc_range*)a;
    const orc_range* y = (const orc_range*)b;
    if (x->begin != y->begin)
        return x->begin < y->begin ? -1 : 1;
    return 0;
}

static int is_pow2(uint64_t x) { return x && !(x & (x - 1)); }

/* Table validity: alignments are powers of two, source ends do not overflow,
 * non-empty source ranges are pairwise disjoint (R8). */
int orc_check(size_t n, const uint64_t* nbytes, const uint64_t* src_offset,
              const uint64_t* dst_align)
{
    for (size_t i = 0; i < n; ++i) {
        if (!is_pow2(dst_align[i]))
            return ORC_EINVAL;
        if (nbytes[i] > UINT64_MAX - src_offset[i])
            return ORC_EOVERFLOW;
    }
    orc_range* r = (orc_range*)malloc((n ? n : 1) * sizeof(orc_range));
    if (!r)
        return ORC_EINVAL;
    size_t m = 0;
    for (size_t i = 0; i < n; ++i)
        if (nbytes[i]) {
            r[m].begin = src_offset[i];
            r[m].end = src_offset[i] + nbytes[i];
            ++m;
        }
    qsort(r, m, sizeof(orc_range), cmp_range);
    int rc = ORC_OK;
    for (size_t j = 1; j < m; ++j)
        if (r[j].begin < r[j - 1].end)
            rc = ORC_EOVERLAP;
    free(r);
    return rc;
}

/* R4: destination offsets in table order and the arena size. */
int orc_layout(size_t n, const uint64_t* nbytes, const uint64_t* dst_align, uint64_t* dst_offset,
               uint64_t* arena_bytes)
{
    uint64_t end = 0, maxal = 1;
    for (size_t i = 0; i < n; ++i) {
        uint64_t a = dst_align[i];
        if (!is_pow2(a))
            return ORC_EINVAL;
        if (end > UINT64_MAX - (a - 1))
            return ORC_EOVERFLOW;
        uint64_t off = (end + a - 1) / a * a;
        if (nbytes[i] > UINT64_MAX - off)
            return ORC_EOVERFLOW;
        dst_offset[i] = off;
        end = off + nbytes[i];
        if (a > maxal)
            maxal = a;
    }
    if (end > UINT64_MAX - (maxal - 1))
        return ORC_EOVERFLOW;
    *arena_bytes = (end + maxal - 1) / maxal * maxal;
    return ORC_OK;
}

/* R1: the span [lo, hi) of the tensors' source bytes (both 0 if every tensor
 * is empty). */
void orc_span(size_t n, const uint64_t* nbytes, const uint64_t* src_offset, uint64_t* lo,
              uint64_t* hi)
{
    uint64_t l = UINT64_MAX, h = 0;
    for (size_t i = 0; i < n; ++i)
        if (nbytes[i]) {
            if (src_offset[i] < l)
                l = src_offset[i];
            if (src_offset[i] + nbytes[i] > h)
                h = src_offset[i] + nbytes[i];
        }
    if (h == 0)
        l = 0;
    *lo = l;
    *hi = h;
}

typedef struct {
    uint64_t chunk_off, tensor_off, len;
    uint32_t tensor;
} orc_seg;

static int cmp_seg(const void* a, const void* b)
{
    const orc_seg* x = (const orc_seg*)a;
    const orc_seg* y = (const orc_seg*)b;
    if (x->chunk_off != y->chunk_off)
        return x->chunk_off < y->chunk_off ? -1 : 1;
    return 0;
}

/*
 * Chunks of equal length chunk_bytes over [lo, hi), the last one partial, and
 * for every chunk the pieces of every tensor whose content falls in it,
 * ordered by position in the chunk.
 *
 * Call with NULL output arrays to get the counts *num_chunks and
 * *num_segments; then call again with arrays of those sizes. Segment s is
 * (chunk, offset in chunk, tensor, offset in tensor, length).
 */
int orc_plan(size_t n, const uint64_t* nbytes, const uint64_t* src_offset, uint64_t chunk_bytes,
             size_t* num_chunks, size_t* num_segments, uint64_t* chunk_begin,
             uint64_t* chunk_len, uint32_t* seg_chunk, uint64_t* seg_chunk_off,
             uint32_t* seg_tensor, uint64_t* seg_tensor_off, uint64_t* seg_len)
{
    if (chunk_bytes == 0)
        return ORC_EINVAL;
    uint64_t lo, hi;
    orc_span(n, nbytes, src_offset, &lo, &hi);
    size_t K = 0;
    for (uint64_t b = lo; b < hi; b += chunk_bytes) {
        if (chunk_begin) {
            chunk_begin[K] = b;
            chunk_len[K] = (hi - b < chunk_bytes) ? hi - b : chunk_bytes;
        }
        ++K;
        if (b > UINT64_MAX - chunk_bytes)
            break;
    }
    *num_chunks = K;

    orc_seg* tmp = (orc_seg*)malloc((n ? n : 1) * sizeof(orc_seg));
    if (!tmp)
        return ORC_EINVAL;
    size_t S = 0;
    for (size_t k = 0; k < K; ++k) {
        uint64_t cb = lo + (uint64_t)k * chunk_bytes;
        uint64_t ce = (hi - cb < chunk_bytes) ? hi : cb + chunk_bytes;
        size_t m = 0;
        for (size_t i = 0; i < n; ++i) {
            if (nbytes[i] == 0)
                continue;
            uint64_t tb = src_offset[i], te = src_offset[i] + nbytes[i];
            uint64_t b = tb > cb ? tb : cb;
            uint64_t e = te < ce ? te : ce;
            if (b < e) {
                tmp[m].chunk_off = b - cb;
                tmp[m].tensor_off = b - tb;
                tmp[m].tensor = (uint32_t)i;
                tmp[m].len = e - b;
                ++m;
            }
        }
        qsort(tmp, m, sizeof(orc_seg), cmp_seg);
        for (size_t j = 0; j < m; ++j, ++S) {
            if (seg_chunk) {
                seg_chunk[S] = (uint32_t)k;
                seg_chunk_off[S] = tmp[j].chunk_off;
                seg_tensor[S] = tmp[j].tensor;
                seg_tensor_off[S] = tmp[j].tensor_off;
                seg_len[S] = tmp[j].len;
            }
        }
    }
    free(tmp);
    *num_segments = S;
    return ORC_OK;
}

/* The sequential loader: tensors one at a time, in table order, each copied
 * from the blob into the caller's buffer out[i] (nbytes[i] bytes). */
int orc_load_into(size_t n, const uint64_t* nbytes, const uint64_t* src_offset,
                  const uint8_t* blob, uint64_t blob_len, uint8_t* const* out)
{
    for (size_t i = 0; i < n; ++i) {
        if (nbytes[i] == 0)
            continue;
        if (src_offset[i] > blob_len || nbytes[i] > blob_len - src_offset[i])
            return ORC_ERANGE;
        memcpy(out[i], blob + src_offset[i], nbytes[i]);
    }
    return ORC_OK;
}

/* The same loader as a plain program would run it: each tensor gets its own
 * freshly allocated buffer (aligned to its dst_align, at least 16 bytes),
 * then its bytes are copied in. out[i] receives the buffer (NULL for empty
 * tensors); release with orc_free. */
int orc_load_alloc(size_t n, const uint64_t* nbytes, const uint64_t* src_offset,
                   const uint64_t* dst_align, const uint8_t* blob, uint64_t blob_len,
                   uint8_t** out)
{
    for (size_t i = 0; i < n; ++i)
        out[i] = NULL;
    for (size_t i = 0; i < n; ++i) {
        if (nbytes[i] == 0)
            continue;
        if (src_offset[i] > blob_len || nbytes[i] > blob_len - src_offset[i])
            return ORC_ERANGE;
        uint64_t a = dst_align[i] < 16 ? 16 : dst_align[i];
        uint64_t sz = (nbytes[i] + a - 1) / a * a;
        out[i] = (uint8_t*)aligned_alloc(a, sz);
        if (!out[i])
            return ORC_EINVAL;
        memcpy(out[i], blob + src_offset[i], nbytes[i]);
    }
    return ORC_OK;
}

void orc_free(size_t n, uint8_t** bufs)
{
    for (size_t i = 0; i < n; ++i) {
        free(bufs[i]);
        bufs[i] = NULL;
    }
}

/* Expected arena after a load into an arena laid out by R4: each tensor's
 * bytes at its destination offset; every other arena byte keeps whatever the
 * caller put there (the canary). */
int orc_arena(size_t n, const uint64_t* nbytes, const uint64_t* src_offset,
              const uint64_t* dst_align, const uint8_t* blob, uint64_t blob_len, uint8_t* arena,
              uint64_t arena_len)
{
    uint64_t* off = (uint64_t*)malloc((n ? n : 1) * sizeof(uint64_t));
    if (!off)
        return ORC_EINVAL;
    uint64_t need;
    int rc = orc_layout(n, nbytes, dst_align, off, &need);
    if (rc == ORC_OK && need > arena_len)
        rc = ORC_ERANGE;
    for (size_t i = 0; rc == ORC_OK && i < n; ++i) {
        if (nbytes[i] == 0)
            continue;
        if (src_offset[i] > blob_len || nbytes[i] > blob_len - src_offset[i]) {
            rc = ORC_ERANGE;
            break;
        }
        memcpy(arena + off[i], blob + src_offset[i], nbytes[i]);
    }
    free(off);
    return rc;
}

/* Expected arena after switching it from the old table's layout to the new
 * one, in place: old tensor ranges are cleared to zero, then every new tensor
 * is written at its new offset. Bytes in a new range end up with new bytes,
 * bytes only in an old range end up zero, all others are untouched. */
int orc_switch(size_t n_old, const uint64_t* nbytes_old, const uint64_t* dst_align_old,
               size_t n_new, const uint64_t* nbytes_new, const uint64_t* src_new,
               const uint64_t* dst_align_new, const uint8_t* blob_new, uint64_t blob_len,
               uint8_t* arena, uint64_t arena_len)
{
    uint64_t* off = (uint64_t*)malloc((n_old ? n_old : 1) * sizeof(uint64_t));
    if (!off)
        return ORC_EINVAL;
    uint64_t need_old;
    int rc = orc_layout(n_old, nbytes_old, dst_align_old, off, &need_old);
    if (rc == ORC_OK && need_old > arena_len)
        rc = ORC_ERANGE;
    for (size_t i = 0; rc == ORC_OK && i < n_old; ++i)
        memset(arena + off[i], 0, nbytes_old[i]);
    free(off);
    if (rc)
        return rc;
    return orc_arena(n_new, nbytes_new, src_new, dst_align_new, blob_new, blob_len, arena,
                     arena_len);
}

/* ---- tensors given as rows (tensor-parallel shards) ------------------- */

/* Rows of each tensor: 0 if it is empty; 1 if its stride is 0 (contiguous);
 * otherwise shape[0] rows of nbytes / shape[0] bytes each, which needs
 * ndim >= 1. */
int orc_rows(size_t n, const int32_t* ndim, const int64_t* shape_flat, const int64_t* shape_start,
             const uint64_t* stride, const uint64_t* nbytes, uint64_t* rows)
{
    for (size_t i = 0; i < n; ++i) {
        if (nbytes[i] == 0) {
            rows[i] = 0;
        } else if (stride[i] == 0) {
            rows[i] = 1;
        } else {
            if (ndim[i] < 1)
                return ORC_EINVAL;
            rows[i] = (uint64_t)shape_flat[shape_start[i]];
        }
    }
    return ORC_OK;
}

/* bytes per row, and the stride actually used (a single row has no stride) */
static uint64_t row_bytes(const uint64_t* nbytes, const uint64_t* rows, size_t i)
{
    return rows[i] ? nbytes[i] / rows[i] : 0;
}

/* Validity: every row fits in 64 bits, rows of one tensor do not overlap
 * each other (stride >= row bytes), and no byte belongs to two rows of any
 * tensors. */
int orc_check_rows(size_t n, const uint64_t* nbytes, const uint64_t* src_offset,
                   const uint64_t* rows, const uint64_t* stride, const uint64_t* dst_align)
{
    size_t total = 0;
    for (size_t i = 0; i < n; ++i) {
        if (!is_pow2(dst_align[i]))
            return ORC_EINVAL;
        if (rows[i] > 1 && stride[i] < row_bytes(nbytes, rows, i))
            return ORC_EINVAL;
        if (rows[i]) {
            uint64_t rb = row_bytes(nbytes, rows, i);
            if (rows[i] > 1 && stride[i] > (UINT64_MAX - src_offset[i]) / (rows[i] - 1))
                return ORC_EOVERFLOW;
            uint64_t last = src_offset[i] + (rows[i] > 1 ? (rows[i] - 1) * stride[i] : 0);
            if (rb > UINT64_MAX - last)
                return ORC_EOVERFLOW;
        }
        total += (size_t)rows[i];
    }
    orc_range* r = (orc_range*)malloc((total ? total : 1) * sizeof(orc_range));
    if (!r)
        return ORC_EINVAL;
    size_t m = 0;
    for (size_t i = 0; i < n; ++i)
        for (uint64_t q = 0; q < rows[i]; ++q) {
            r[m].begin = src_offset[i] + q * stride[i];
            r[m].end = r[m].begin + row_bytes(nbytes, rows, i);
            ++m;
        }
    qsort(r, m, sizeof(orc_range), cmp_range);
    int rc = ORC_OK;
    for (size_t j = 1; j < m; ++j)
        if (r[j].begin < r[j - 1].end)
            rc = ORC_EOVERLAP;
    free(r);
    return rc;
}

/* R1 for rows: from the first byte of any row to the end of the last. */
void orc_span_rows(size_t n, const uint64_t* nbytes, const uint64_t* src_offset,
                   const uint64_t* rows, const uint64_t* stride, uint64_t* lo, uint64_t* hi)
{
    uint64_t l = UINT64_MAX, h = 0;
    for (size_t i = 0; i < n; ++i)
        for (uint64_t q = 0; q < rows[i]; ++q) {
            uint64_t b = src_offset[i] + q * stride[i];
            uint64_t e = b + row_bytes(nbytes, rows, i);
            if (b < l)
                l = b;
            if (e > h)
                h = e;
        }
    if (h == 0)
        l = 0;
    *lo = l;
    *hi = h;
}

/* orc_plan for rows: every row of every tensor cut at chunk boundaries; a
 * piece's offset in its tensor is (row index x row bytes) + its offset in the
 * row. Same two-call protocol as orc_plan. */
int orc_plan_rows(size_t n, const uint64_t* nbytes, const uint64_t* src_offset,
                  const uint64_t* rows, const uint64_t* stride, uint64_t chunk_bytes,
                  size_t* num_chunks, size_t* num_segments, uint64_t* chunk_begin,
                  uint64_t* chunk_len, uint32_t* seg_chunk, uint64_t* seg_chunk_off,
                  uint32_t* seg_tensor, uint64_t* seg_tensor_off, uint64_t* seg_len)
{
    if (chunk_bytes == 0)
        return ORC_EINVAL;
    uint64_t lo, hi;
    orc_span_rows(n, nbytes, src_offset, rows, stride, &lo, &hi);
    size_t K = 0;
    for (uint64_t b = lo; b < hi; b += chunk_bytes) {
        if (chunk_begin) {
            chunk_begin[K] = b;
            chunk_len[K] = (hi - b < chunk_bytes) ? hi - b : chunk_bytes;
        }
        ++K;
        if (b > UINT64_MAX - chunk_bytes)
            break;
    }
    *num_chunks = K;
    size_t total = 0;
    for (size_t i = 0; i < n; ++i)
        total += (size_t)rows[i];
    orc_seg* tmp = (orc_seg*)malloc((total ? total : 1) * sizeof(orc_seg));
    if (!tmp)
        return ORC_EINVAL;
    size_t S = 0;
    for (size_t k = 0; k < K; ++k) {
        uint64_t cb = lo + (uint64_t)k * chunk_bytes;
        uint64_t ce = (hi - cb < chunk_bytes) ? hi : cb + chunk_bytes;
        size_t m = 0;
        for (size_t i = 0; i < n; ++i) {
            uint64_t rb = row_bytes(nbytes, rows, i);
            for (uint64_t q = 0; q < rows[i]; ++q) {
                uint64_t rs = src_offset[i] + q * stride[i], re = rs + rb;
                uint64_t b = rs > cb ? rs : cb;
                uint64_t e = re < ce ? re : ce;
                if (b < e) {
                    tmp[m].chunk_off = b - cb;
                    tmp[m].tensor_off = q * rb + (b - rs);
                    tmp[m].tensor = (uint32_t)i;
                    tmp[m].len = e - b;
                    ++m;
                }
            }
        }
        qsort(tmp, m, sizeof(orc_seg), cmp_seg);
        for (size_t j = 0; j < m; ++j, ++S) {
            if (seg_chunk) {
                seg_chunk[S] = (uint32_t)k;
                seg_chunk_off[S] = tmp[j].chunk_off;
                seg_tensor[S] = tmp[j].tensor;
                seg_tensor_off[S] = tmp[j].tensor_off;
                seg_len[S] = tmp[j].len;
            }
        }
    }
    free(tmp);
    *num_segments = S;
    return ORC_OK;
}

/* The sequential loader for rows: tensor by tensor, row by row, each row
 * appended to the tensor's buffer. */
int orc_load_rows_into(size_t n, const uint64_t* nbytes, const uint64_t* src_offset,
                       const uint64_t* rows, const uint64_t* stride, const uint8_t* blob,
                       uint64_t blob_len, uint8_t* const* out)
{
    for (size_t i = 0; i < n; ++i) {
        uint64_t rb = row_bytes(nbytes, rows, i);
        for (uint64_t q = 0; q < rows[i]; ++q) {
            uint64_t s = src_offset[i] + q * stride[i];
            if (s > blob_len || rb > blob_len - s)
                return ORC_ERANGE;
            memcpy(out[i] + q * rb, blob + s, rb);
        }
    }
    return ORC_OK;
}

/* Expected arena after a load of a table given as rows (layout R4). */
int orc_arena_rows(size_t n, const uint64_t* nbytes, const uint64_t* src_offset,
                   const uint64_t* rows, const uint64_t* stride, const uint64_t* dst_align,
                   const uint8_t* blob, uint64_t blob_len, uint8_t* arena, uint64_t arena_len)
{
    uint64_t* off = (uint64_t*)malloc((n ? n : 1) * sizeof(uint64_t));
    uint8_t** out = (uint8_t**)malloc((n ? n : 1) * sizeof(uint8_t*));
    if (!off || !out) {
        free(off);
        free(out);
        return ORC_EINVAL;
    }
    uint64_t need;
    int rc = orc_layout(n, nbytes, dst_align, off, &need);
    if (rc == ORC_OK && need > arena_len)
        rc = ORC_ERANGE;
    if (rc == ORC_OK) {
        for (size_t i = 0; i < n; ++i)
            out[i] = arena + off[i];
        rc = orc_load_rows_into(n, nbytes, src_offset, rows, stride, blob, blob_len, out);
    }
    free(off);
    free(out);
    return rc;
}
