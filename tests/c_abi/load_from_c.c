/*
 * A plain C user of libii.so: no Python, no PyTorch. Builds a small
 * transformer-shaped table in memory (4 layers, hidden 256, FFN 1024, vocab
 * 8192, bf16), fills a blob with a counter-based pattern, plans with 1 MiB
 * chunks, loads into one device arena on its own stream, copies the arena
 * back and checks every tensor byte against the blob and every padding byte
 * against its fill value. Prints "OK <tensors> <bytes>" and exits 0 on
 * success.
 *
 * Device memory, the stream and the copies use the HIP runtime directly.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "ii.h"

/* the few HIP runtime calls this program needs, declared by hand so that it
 * builds without the ROCm headers */
typedef int hipError_t;
hipError_t hipMalloc(void** p, size_t n);
hipError_t hipFree(void* p);
hipError_t hipMemset(void* p, int v, size_t n);
hipError_t hipMemcpy(void* dst, const void* src, size_t n, int kind);
hipError_t hipStreamCreate(hipStream_t* s);
hipError_t hipStreamSynchronize(hipStream_t s);
hipError_t hipStreamDestroy(hipStream_t s);
enum { kD2H = 2 };

#define DIE(...) do { fprintf(stderr, __VA_ARGS__); fprintf(stderr, "\n"); return 1; } while (0)

int main(void) {
    enum { L = 4, H = 256, F = 1024, V = 8192, N = 1 + 9 * L + 2 };
    static int64_t shapes[N][2];
    static int32_t ndims[N];
    ii_tensor_desc t[N];
    int i = 0;
    shapes[i][0] = V; shapes[i][1] = H; ndims[i++] = 2;              /* embed */
    for (int l = 0; l < L; ++l) {
        const int64_t s[9][2] = {{H, 0}, {H, H}, {H, H}, {H, H}, {H, H}, {H, 0}, {F, H}, {F, H}, {H, F}};
        for (int j = 0; j < 9; ++j) {
            shapes[i][0] = s[j][0]; shapes[i][1] = s[j][1];
            ndims[i++] = s[j][1] ? 2 : 1;
        }
    }
    shapes[i][0] = H; ndims[i++] = 1;                                 /* final norm */
    shapes[i][0] = V; shapes[i][1] = H; ndims[i++] = 2;              /* lm_head */
    uint64_t pos = 4096;                                              /* a header before the tensors */
    for (i = 0; i < N; ++i) {
        uint64_t nb = 2;
        for (int d = 0; d < ndims[i]; ++d) nb *= (uint64_t)shapes[i][d];
        t[i].name = NULL;
        t[i].dtype = II_BF16;
        t[i].ndim = ndims[i];
        t[i].shape = shapes[i];
        t[i].src_offset = pos;
        t[i].dst_align = (i % 2) ? 256 : 4096;
        t[i].src_row_stride = 0;                                      /* contiguous */
        pos += nb + 8;                                                /* small gaps in the file */
    }
    const uint64_t blob_bytes = pos;
    uint8_t* blob = malloc(blob_bytes);
    if (!blob) DIE("malloc");
    for (uint64_t x = 0; x < blob_bytes; ++x) blob[x] = (uint8_t)((x * 2654435761u) >> 11);

    ii_plan_t* plan = NULL;
    int rc = ii_plan(t, N, 1u << 20, &plan);
    if (rc) DIE("ii_plan: %s (%s)", ii_strerror(rc), ii_last_error());
    const uint64_t arena_bytes = ii_plan_arena_bytes(plan);
    uint64_t nbytes[N], off[N];
    ii_plan_tensors(plan, nbytes, off);

    uint8_t* arena = NULL;
    if (hipMalloc((void**)&arena, arena_bytes)) DIE("hipMalloc");
    if (hipMemset(arena, 0x5A, arena_bytes)) DIE("hipMemset");
    void* dst[N];
    for (i = 0; i < N; ++i) dst[i] = arena + off[i];
    hipStream_t s;
    if (hipStreamCreate(&s)) DIE("hipStreamCreate");
    rc = ii_load(plan, blob, blob_bytes, dst, s);
    if (rc) DIE("ii_load: %s (%s)", ii_strerror(rc), ii_last_error());
    if (hipStreamSynchronize(s)) DIE("hipStreamSynchronize");

    uint8_t* back = malloc(arena_bytes);
    if (!back || hipMemcpy(back, arena, arena_bytes, kD2H)) DIE("readback");
    uint8_t* want = malloc(arena_bytes);
    memset(want, 0x5A, arena_bytes);
    uint64_t payload = 0;
    for (i = 0; i < N; ++i) {
        memcpy(want + off[i], blob + t[i].src_offset, nbytes[i]);
        payload += nbytes[i];
    }
    if (memcmp(back, want, arena_bytes)) {
        for (uint64_t x = 0; x < arena_bytes; ++x)
            if (back[x] != want[x]) DIE("mismatch at arena byte %llu", (unsigned long long)x);
    }
    ii_plan_free(plan);
    hipStreamDestroy(s);
    hipFree(arena);
    free(blob);
    free(back);
    free(want);
    printf("OK %d %llu\n", N, (unsigned long long)payload);
    return 0;
}
