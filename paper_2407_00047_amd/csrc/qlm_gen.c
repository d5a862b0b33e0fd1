/*
 * qlm_gen.c -- seeded synthetic candidate plans for QLM plan scoring.
 *
 * Input generation only: no waiting-time, probability or scoring arithmetic.
 * Both the HIP path and the CPU oracle read what this writes.
 *
 * A plan (Sec. 7 of arXiv 2407.00047: each request group takes exactly one
 * position in exactly one virtual queue, Eq. slot_assignment) is drawn as
 *   1. an independent uniform queue for every group (when there is more than
 *      one queue),
 *   2. a uniformly random order of the groups within each queue,
 *   3. optionally exactly n_evict distinct slots flagged for eviction.
 * Plan p uses its own random stream, so any subrange of plans can be
 * regenerated alone.
 *
 * Generators (named, published, written here from their definitions):
 *   splitmix64 (Steele, Lea, Flood 2014) to seed,
 *   xoshiro256** (Blackman, Vigna 2018) for the stream,
 *   Lemire's nearly divisionless bounded integers (2019),
 *   Fisher-Yates shuffle, Floyd's sampling of distinct values.
 *
 * Output layout is slot-major with plan stride ld (elements):
 *   perm[s*ld + p], qoff[g*ld + p] (g = 0..I), evict[w*ld + p] (w = 0..ceil(G/32)-1).
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

typedef struct { uint64_t s[4]; } rng_t;

static uint64_t splitmix64(uint64_t *x)
{
    uint64_t z = (*x += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

static uint64_t rotl(uint64_t x, int k) { return (x << k) | (x >> (64 - k)); }

static uint64_t next64(rng_t *r)
{
    uint64_t *s = r->s;
    const uint64_t result = rotl(s[1] * 5, 7) * 9;
    const uint64_t t = s[1] << 17;
    s[2] ^= s[0];
    s[3] ^= s[1];
    s[1] ^= s[2];
    s[0] ^= s[3];
    s[2] ^= t;
    s[3] = rotl(s[3], 45);
    return result;
}

static void seed_plan(rng_t *r, uint64_t seed, int64_t plan)
{
    uint64_t x = seed ^ ((uint64_t)plan * 0xD1B54A32D192ED03ull);
    for (int k = 0; k < 4; ++k) r->s[k] = splitmix64(&x);
}

/* uniform integer in [0, range), range >= 1 (Lemire 2019) */
static uint32_t bounded(rng_t *r, uint32_t range)
{
    uint32_t x = (uint32_t)(next64(r) >> 32);
    uint64_t m = (uint64_t)x * range;
    uint32_t l = (uint32_t)m;
    if (l < range) {
        uint32_t t = (uint32_t)(-range) % range;
        while (l < t) {
            x = (uint32_t)(next64(r) >> 32);
            m = (uint64_t)x * range;
            l = (uint32_t)m;
        }
    }
    return (uint32_t)(m >> 32);
}

/* One plan into plan-contiguous scratch: perm[G], qoff[I+1], ev[W]. */
static void one_plan(uint64_t seed, int64_t p, int G, int I, int n_evict,
                     int32_t *perm, int32_t *qoff, uint32_t *ev,
                     int32_t *order, int32_t *owner, int32_t *fill)
{
    rng_t r;
    seed_plan(&r, seed, p);
    for (int i = 0; i < G; ++i) order[i] = i;
    for (int i = G - 1; i > 0; --i) {             /* Fisher-Yates */
        int j = (int)bounded(&r, (uint32_t)i + 1u);
        int32_t t = order[i]; order[i] = order[j]; order[j] = t;
    }
    if (I == 1) {
        memcpy(perm, order, sizeof(int32_t) * (size_t)G);
        qoff[0] = 0; qoff[1] = G;
    } else {
        for (int g = 0; g <= I; ++g) qoff[g] = 0;
        for (int i = 0; i < G; ++i) {
            owner[i] = (int32_t)bounded(&r, (uint32_t)I);
            qoff[owner[i] + 1] += 1;
        }
        for (int g = 0; g < I; ++g) qoff[g + 1] += qoff[g];
        for (int g = 0; g < I; ++g) fill[g] = qoff[g];
        for (int k = 0; k < G; ++k) {                /* groups in shuffled order */
            int i = order[k];
            perm[fill[owner[i]]++] = i;
        }
    }
    const int W = (G + 31) / 32;
    if (ev) {
        for (int w = 0; w < W; ++w) ev[w] = 0u;
        /* Floyd: n_evict distinct slots out of G */
        for (int j = G - n_evict; j < G; ++j) {
            int t = (int)bounded(&r, (uint32_t)j + 1u);
            if (ev[t / 32] & (1u << (t % 32))) t = j;
            ev[t / 32] |= 1u << (t % 32);
        }
    }
}

/* Plans [p0, p0+count) written at columns [0, count) of the output arrays.
 * evict may be NULL (then n_evict is ignored).  Returns 0, or -1 on bad sizes. */
int qlm_gen_plans(uint64_t seed, int64_t p0, int64_t count, int G, int I, int n_evict,
                  int64_t ld, int32_t *perm, int32_t *qoff, uint32_t *evict, int n_threads)
{
    enum { BLK = 16 };
    if (G < 1 || I < 1 || count < 0 || ld < count || (evict && (n_evict < 0 || n_evict > G)))
        return -1;
    const int W = (G + 31) / 32;
    const int64_t nblk = (count + BLK - 1) / BLK;
    int err = 0;
#ifdef _OPENMP
    if (n_threads <= 0) n_threads = omp_get_max_threads();
#pragma omp parallel num_threads(n_threads) reduction(| : err)
#endif
    {
        int32_t *bp = malloc(sizeof(int32_t) * (size_t)G * BLK);
        int32_t *bq = malloc(sizeof(int32_t) * (size_t)(I + 1) * BLK);
        uint32_t *be = malloc(sizeof(uint32_t) * (size_t)W * BLK);
        int32_t *order = malloc(sizeof(int32_t) * (size_t)G);
        int32_t *owner = malloc(sizeof(int32_t) * (size_t)G);
        int32_t *fill = malloc(sizeof(int32_t) * (size_t)I);
        if (!bp || !bq || !be || !order || !owner || !fill) {
            err = 1;
        } else {
#ifdef _OPENMP
#pragma omp for schedule(dynamic, 4)
#endif
            for (int64_t b = 0; b < nblk; ++b) {
                const int64_t c0 = b * BLK;
                const int nb = (int)((count - c0) < BLK ? (count - c0) : BLK);
                for (int k = 0; k < nb; ++k)
                    one_plan(seed, p0 + c0 + k, G, I, n_evict, bp + (size_t)k * G,
                             bq + (size_t)k * (I + 1), evict ? be + (size_t)k * W : NULL,
                             order, owner, fill);
                /* transpose the block into the slot-major outputs */
                for (int s = 0; s < G; ++s)
                    for (int k = 0; k < nb; ++k)
                        perm[(int64_t)s * ld + c0 + k] = bp[(size_t)k * G + s];
                for (int g = 0; g <= I; ++g)
                    for (int k = 0; k < nb; ++k)
                        qoff[(int64_t)g * ld + c0 + k] = bq[(size_t)k * (I + 1) + g];
                if (evict)
                    for (int w = 0; w < W; ++w)
                        for (int k = 0; k < nb; ++k)
                            evict[(int64_t)w * ld + c0 + k] = be[(size_t)k * W + w];
            }
        }
        free(bp); free(bq); free(be); free(order); free(owner); free(fill);
    }
    (void)n_threads;
    return err ? -1 : 0;
}
