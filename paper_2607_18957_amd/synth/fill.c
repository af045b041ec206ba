/*
 * Seeded blob filler for the synthetic weight sets.
 *
 * The blob stands in for a checkpoint file's bytes held in host memory. Its
 * contents are a counter-based stream: the little-endian 64-bit word at blob
 * offset 8*j is splitmix64(seed * 2^40 + j), where splitmix64(x) is the output
 * of one step of Steele, Lea and Flood's SplitMix64 generator ("Fast
 * splittable pseudorandom number generators", OOPSLA 2014) started from state
 * x: add the golden-ratio increment, then apply the variant-13 finaliser.
 * Any byte can therefore be regenerated on its own, and the fill runs in
 * parallel over disjoint ranges.
 *
 * This file generates inputs only. It holds none of the loader's arithmetic
 * and is shared by the oracle-side and device-side tests as the common input
 * source.
 */
#include <pthread.h>
#include <stdint.h>
#include <string.h>

static inline uint64_t sm64(uint64_t x)
{
    uint64_t z = x + 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

/* The blob word with index j for the given seed. */
uint64_t synth_word(uint64_t seed, uint64_t j)
{
    return sm64((seed << 40) + j);
}

/* Fill dst[0, len) with blob bytes [offset, offset + len). Single thread. */
static void fill_range(uint8_t* dst, uint64_t offset, uint64_t len, uint64_t seed)
{
    uint64_t base = seed << 40;
    uint64_t x = offset;
    uint64_t end = offset + len;
    /* leading bytes up to the next word boundary */
    while (x < end && (x & 7u)) {
        uint64_t w = sm64(base + (x >> 3));
        dst[x - offset] = (uint8_t)(w >> (8u * (x & 7u)));
        ++x;
    }
    /* whole words */
    while (x + 8 <= end) {
        uint64_t w = sm64(base + (x >> 3));
        memcpy(dst + (x - offset), &w, 8); /* host is little-endian (x86-64) */
        x += 8;
    }
    /* trailing bytes */
    while (x < end) {
        uint64_t w = sm64(base + (x >> 3));
        dst[x - offset] = (uint8_t)(w >> (8u * (x & 7u)));
        ++x;
    }
}

typedef struct {
    uint8_t* dst;
    uint64_t offset, len, seed;
} fill_job;

static void* fill_worker(void* arg)
{
    fill_job* j = (fill_job*)arg;
    fill_range(j->dst, j->offset, j->len, j->seed);
    return NULL;
}

/* Fill dst[0, len) with blob bytes [offset, offset + len) using up to
 * `threads` threads (1..256). Returns 0 on success, -1 on a bad argument. */
int synth_fill(uint8_t* dst, uint64_t offset, uint64_t len, uint64_t seed, int threads)
{
    if (!dst && len)
        return -1;
    if (threads < 1)
        threads = 1;
    if (threads > 256)
        threads = 256;
    if (len < (1u << 22) || threads == 1) {
        fill_range(dst, offset, len, seed);
        return 0;
    }
    pthread_t tid[256];
    fill_job jobs[256];
    uint64_t per = (len / (uint64_t)threads + 4095u) & ~(uint64_t)4095u;
    int started = 0;
    for (int t = 0; t < threads; ++t) {
        uint64_t b = (uint64_t)t * per;
        if (b >= len)
            break;
        uint64_t e = b + per < len ? b + per : len;
        jobs[t].dst = dst + b;
        jobs[t].offset = offset + b;
        jobs[t].len = e - b;
        jobs[t].seed = seed;
        if (pthread_create(&tid[t], NULL, fill_worker, &jobs[t]) != 0) {
            fill_range(jobs[t].dst, jobs[t].offset, jobs[t].len, seed);
            jobs[t].len = 0;
            tid[t] = 0;
        }
        started = t + 1;
    }
    for (int t = 0; t < started; ++t)
        if (tid[t])
            pthread_join(tid[t], NULL);
    return 0;
}
