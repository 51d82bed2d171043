/* CPU check of the oracle under AddressSanitizer and UndefinedBehaviorSanitizer
 * (built by tests/test_sanitize.py, with and without the sanitizers): rounds
 * of every update rule and local optimizer, with and without lost messages,
 * on chains, stars and random trees of 1 to 40 workers, in float and double.
 * Prints one FNV-1a digest of every output bit; the sanitized and the plain
 * build must print the same digest. */
#include <stdio.h>
#include <stdlib.h>

#include "../../oracle/relaysum_oracle.c"

static unsigned long long digest = 1469598103934665603ull;
static void mix(const void *p, size_t bytes) {
    const unsigned char *c = (const unsigned char *)p;
    for (size_t k = 0; k < bytes; ++k) {
        digest ^= c[k];
        digest *= 1099511628211ull;
    }
}

static unsigned long long rng = 88172645463325252ull;
static unsigned long long next_u64(void) {
    rng ^= rng << 13;
    rng ^= rng >> 7;
    rng ^= rng << 17;
    return rng;
}
static double uniform(void) { return (double)(next_u64() >> 11) / 9007199254740992.0; }

/* Tree on n workers: 0 = chain, 1 = star, 2 = random (each worker's parent
 * drawn among the earlier ones). */
static void tree(int n, int kind, int *edges) {
    for (int i = 1; i < n; ++i) {
        edges[2 * (i - 1)] = kind == 0 ? i - 1 : kind == 1 ? 0 : (int)(next_u64() % (unsigned)i);
        edges[2 * (i - 1) + 1] = i;
    }
}

#define RUN(P, REALT)                                                                       \
    static void run_##P(int n, int64_t d, int kind, int update, int optimizer, double p_drop) { \
        int *edges = malloc(sizeof(int) * 2 * (n > 1 ? n - 1 : 1));                        \
        tree(n, kind, edges);                                                               \
        void *h = oracle_##P##_create(n, d, n - 1, edges);                                  \
        REALT *x = calloc((size_t)(n * d) + 1, sizeof(REALT));                              \
        REALT *g = calloc((size_t)(n * d) + 1, sizeof(REALT));                              \
        REALT *s1 = calloc((size_t)(n * d) + 1, sizeof(REALT));                             \
        REALT *s2 = calloc((size_t)(n * d) + 1, sizeof(REALT));                             \
        unsigned char *drop = calloc((size_t)n * n, 1);                                     \
        for (int64_t k = 0; k < n * d; ++k) x[k] = (REALT)(uniform() * 2 - 1);              \
        for (int t = 0; t < 6; ++t) {                                                       \
            for (int64_t k = 0; k < n * d; ++k) g[k] = (REALT)(uniform() * 2 - 1);          \
            for (int k = 0; k < n * n; ++k) drop[k] = uniform() < p_drop;                  \
            const REALT beta1 = optimizer == 1 ? (REALT)0.9 : update >= 2 ? 0 : (REALT)0.5;  \
            oracle_##P##_round_ex(h, x, g, s1, s2, update, optimizer, (REALT)0.05, beta1,   \
                                  (REALT)0.999, (REALT)1e-8, t + 1, p_drop > 0 ? drop : NULL); \
            mix(x, sizeof(REALT) * (size_t)(n * d));                                        \
            mix(s1, sizeof(REALT) * (size_t)(n * d));                                       \
            for (int i = 0; i < n; ++i) {                                                   \
                const int nb = oracle_##P##_nbar(h, i);                                     \
                const long long sm = (long long)oracle_##P##_samples(h, i);                 \
                mix(&nb, sizeof nb);                                                        \
                mix(&sm, sizeof sm);                                                        \
            }                                                                               \
        }                                                                                   \
        oracle_##P##_destroy(h);                                                            \
        free(edges); free(x); free(g); free(s1); free(s2); free(drop);                      \
    }
RUN(f32, float)
RUN(f64, double)

int main(void) {
    static const int sizes[] = {1, 2, 3, 5, 9, 16, 40};
    static const int64_t dims[] = {1, 3, 17};
    for (size_t a = 0; a < sizeof sizes / sizeof *sizes; ++a)
        for (size_t b = 0; b < sizeof dims / sizeof *dims; ++b)
            for (int kind = 0; kind < 3; ++kind)
                for (int update = 0; update < 4; ++update)
                    for (int optimizer = 0; optimizer < 2; ++optimizer) {
                        if (optimizer == 1 && update >= 2) continue;
                        for (int drops = 0; drops < 2; ++drops) {
                            run_f32(sizes[a], dims[b], kind, update, optimizer, drops ? 0.2 : 0.0);
                            run_f64(sizes[a], dims[b], kind, update, optimizer, drops ? 0.2 : 0.0);
                        }
                    }
    printf("digest %016llx\n", digest);
    return 0;
}
