/* RelaySum oracle: a plain, slow CPU implementation of one RelaySGD round
 * (Alg. 1 of the paper, with the Nesterov local step of Appendix D.2).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; only the tests, the smoke check and the benchmark's CPU
 * baseline do.  It shares no code, header or table with the HIP path.
 *
 * The round is written twice from one source (relaysum_round.inc): in float
 * (binary32, the precision of the fp32 parameter vectors the workloads fix,
 * and the one parity is judged in) and in double (a cross-precision check of
 * the float version).  The loops over coordinates may run on several OpenMP
 * threads; coordinates are independent, so the result does not depend on the
 * thread count.
 *
 * Build: gcc -O2 -ffp-contract=off -fno-fast-math -fopenmp -shared -fPIC
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define REAL float
#define SQRT sqrtf
#define STATE state_f32
#define FN(name) f32_##name
#include "relaysum_round.inc"
#undef REAL
#undef SQRT
#undef STATE
#undef FN

#define REAL double
#define SQRT sqrt
#define STATE state_f64
#define FN(name) f64_##name
#include "relaysum_round.inc"
#undef REAL
#undef SQRT
#undef STATE
#undef FN

/* ---- exported API (two copies, one per precision) ---- */
#define EXPORTS(P, REALT, ST)                                                        \
    void *oracle_##P##_create(int n, int64_t d, int num_edges, const int *edges)    \
    { return (void *)P##_create(n, d, num_edges, edges); }                          \
    void oracle_##P##_destroy(void *h) { P##_free_state((struct ST *)h); }          \
    void oracle_##P##_reset(void *h) { P##_reset((struct ST *)h); }                 \
    int oracle_##P##_round(void *h, REALT *x, const REALT *g, REALT *mom,           \
                           REALT lr, REALT beta)                                    \
    { return P##_round((struct ST *)h, x, g, mom, lr, beta); }                      \
    int oracle_##P##_round_ex(void *h, REALT *x, const REALT *g, REALT *s1, REALT *s2,  \
                              int update, int optimizer, REALT lr, REALT beta1,     \
                              REALT beta2, REALT eps, int64_t adam_t,               \
                              const unsigned char *dropped)                         \
    { return P##_round_ex((struct ST *)h, x, g, s1, s2, update, optimizer, lr,      \
                          beta1, beta2, eps, adam_t, dropped); }                    \
    /* mean estimation: s_i, samples summed into worker i's y_i so far */          \
    int64_t oracle_##P##_samples(void *h, int i)                                    \
    {                                                                               \
        struct ST *s = (struct ST *)h;                                              \
        return (i < 0 || i >= s->n || !s->samples) ? 0 : s->samples[i];             \
    }                                                                               \
    int64_t oracle_##P##_rounds(void *h) { return ((struct ST *)h)->t; }            \
    /* c_{src->dst} sent in the last round; -1 if src,dst are not adjacent */       \
    int oracle_##P##_count(void *h, int src, int dst)                               \
    {                                                                               \
        struct ST *s = (struct ST *)h;                                              \
        if (src < 0 || dst < 0 || src >= s->n || dst >= s->n) return -1;            \
        if (!s->m_prev[src * s->n + dst]) return -1;                                \
        return s->c_prev[src * s->n + dst];                                         \
    }                                                                               \
    /* nbar_i used in the last round's average */                                   \
    int oracle_##P##_nbar(void *h, int i)                                           \
    {                                                                               \
        struct ST *s = (struct ST *)h;                                              \
        return (i < 0 || i >= s->n) ? -1 : s->nbar[i];                              \
    }                                                                               \
    /* m_{src->dst} sent in the last round, d values into out */                    \
    int oracle_##P##_message(void *h, int src, int dst, REALT *out)                 \
    {                                                                               \
        struct ST *s = (struct ST *)h;                                              \
        if (src < 0 || dst < 0 || src >= s->n || dst >= s->n) return -1;            \
        const REALT *m = s->m_prev[src * s->n + dst];                               \
        if (!m) return -1;                                                          \
        memcpy(out, m, sizeof(REALT) * (size_t)s->d);                               \
        return 0;                                                                   \
    }

EXPORTS(f32, float, state_f32)
EXPORTS(f64, double, state_f64)

void oracle_set_threads(int k)
{
#ifdef _OPENMP
    if (k > 0) omp_set_num_threads(k);
#else
    (void)k;
#endif
}

int oracle_get_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
