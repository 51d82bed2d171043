/* relaysum.h -- one synchronous RelaySum round of RelaySGD for all n workers
 * of a tree, simulated on one MI355X (gfx950) GPU.
 *
 * What a round computes (the paper's Alg. 1, "RelaySum/Model", with the
 * Nesterov local step of Appendix D.2).  For round t and every worker i,
 * with N_i the neighbours of i in the tree:
 *
 *   local step   b_i   <- beta*b_i + g_i                         (beta != 0)
 *                xh_i   = x_i - lr*(g_i + beta*b_i)              (beta != 0)
 *                xh_i   = x_i - lr*g_i                           (beta == 0)
 *   relay        m_{i->j}^{(t)} = xh_i + sum_{k in N_i\j} m_{k->i}^{(t-1)}
 *                c_{i->j}^{(t)} = 1    + sum_{k in N_i\j} c_{k->i}^{(t-1)}
 *   average      nbar_i = 1 + sum_{j in N_i} c_{j->i}^{(t)}
 *                x_i    = (xh_i + sum_{j in N_i} m_{j->i}^{(t)}) / nbar_i
 *
 * with m^{(-1)} = 0 and c^{(-1)} = 0 before the first round.  All arithmetic
 * is IEEE binary32, one rounding per operation, no fused multiply-add; every
 * sum over a neighbour set starts from xh_i and adds neighbours in ascending
 * id; the average is a true division.  The result is therefore a fixed
 * function of the inputs (it does not depend on the launch shape).
 *
 * Memory: x, g, mom are DEVICE pointers to row-major float[n][d] (row i is
 * worker i, row stride d floats); they belong to the caller and must not
 * alias each other or any buffer of the handle.  Edge lists and every
 * *_host buffer are HOST memory.  The handle owns the tree (CSR form), a
 * two-slot ring of 2(n-1) messages of d floats each, the integer counters,
 * and the round number.
 *
 * Streams: all device work of a handle is queued on its stream (the null
 * stream until relaysum_set_stream); calls return before that work ends,
 * except the accessors marked "synchronises".  A handle is not thread-safe.
 *
 * Errors: every int-returning function returns RELAYSUM_OK (0) or a negative
 * relaysum_status; relaysum_strerror() names a code and
 * relaysum_last_error() gives the text of the handle's last failure.
 */
#ifndef RELAYSUM_H
#define RELAYSUM_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct relaysum_s relaysum_t;

typedef enum relaysum_status {
    RELAYSUM_OK = 0,
    RELAYSUM_ERR_INVALID_ARG = -1,   /* bad size, NULL pointer, misuse */
    RELAYSUM_ERR_NOT_A_TREE = -2,    /* edge list is not a tree on n workers */
    RELAYSUM_ERR_OUT_OF_MEMORY = -3, /* device or host allocation failed */
    RELAYSUM_ERR_DEVICE = -4         /* HIP runtime or launch error */
} relaysum_status;

/* Create a handle for n workers with d-float models on the tree given by
 * num_edges undirected edges edges[2e], edges[2e+1] (0-based worker ids,
 * HOST memory, any order).  The tree is the paper's communication graph
 * (Section 3, Setup: n >= 1 workers, no self loops); RelaySum needs it to be
 * a tree (Alg. 1 input).
 *   n >= 1, d >= 0 (d == 0: rounds only relay the counters).
 *   Returns RELAYSUM_ERR_NOT_A_TREE unless num_edges == n-1, every id is in
 *   [0, n), and the edges have no self loop, no duplicate and connect all
 *   workers; RELAYSUM_ERR_INVALID_ARG for n < 1, d < 0, out == NULL, or
 *   edges == NULL with num_edges > 0; RELAYSUM_ERR_OUT_OF_MEMORY when device
 *   memory for 2 * 2(n-1) * d floats cannot be had.
 * Allocates on the current HIP device, zeroes every message and counter
 * (m^{(-1)} = 0, c^{(-1)} = 0) and sets the round number to 0.  On failure
 * *out is set to NULL. */
int relaysum_create(int32_t n, int64_t d, const int32_t *edges, int32_t num_edges,
                    relaysum_t **out);

/* Release the handle after waiting for its stream.  NULL is a no-op. */
int relaysum_destroy(relaysum_t *h);

/* Queue later device work on `hip_stream` (a hipStream_t; NULL = null
 * stream).  The caller keeps the stream alive while the handle uses it. */
int relaysum_set_stream(relaysum_t *h, void *hip_stream);

/* One round t (Alg. 1 loop body, all workers), then t <- t+1.
 *   x    [n][d] device, read and overwritten with x^{(t+1)};
 *   g    [n][d] device, read only: the gradients at x^{(t)};
 *   mom  [n][d] device, the Nesterov buffers b_i (start them at 0), updated
 *        in place; may be NULL if and only if beta == 0, and is neither read
 *        nor written when beta == 0;
 *   lr   the learning rate gamma (lr == 0 is allowed: mom still updates);
 *   beta the momentum parameter alpha of Appendix D.2 (0 = plain SGD).
 * Rows must be 4-byte aligned; 16-byte aligned pointers with d % 4 == 0 use
 * 128-bit accesses (same results, faster).
 * Returns RELAYSUM_ERR_INVALID_ARG for h, x or g NULL (unless d == 0), mom
 * NULL with beta != 0, or misaligned pointers; RELAYSUM_ERR_DEVICE if the
 * launch fails (then the round number is not advanced). */
int relaysum_step(relaysum_t *h, float *x, const float *g, float *mom, float lr, float beta);

/* Back to the state before the first round: messages and counters zeroed
 * (queued on the handle's stream), round number 0. */
int relaysum_reset(relaysum_t *h);

/* Number of rounds done since create or reset. */
int relaysum_round(const relaysum_t *h, int64_t *t);

/* Number of directed edges, 2(n-1).  Directed edge "slots" 0..2(n-1)-1 are
 * ordered by source worker, then by destination, ascending. */
int relaysum_num_directed_edges(const relaysum_t *h, int32_t *count);

/* Source and destination worker of a slot (host-side table lookup). */
int relaysum_directed_edge(const relaysum_t *h, int32_t slot, int32_t *src, int32_t *dst);

/* Counters of the last round (synchronises the handle's stream):
 * nbar_host[n] = nbar_i used in the last average, edge_counts_host[2(n-1)]
 * = c_{src->dst} per slot.  Either pointer may be NULL.  Before any round
 * every value is 0. */
int relaysum_get_counts(relaysum_t *h, int32_t *nbar_host, int32_t *edge_counts_host);

/* The d floats of message m_{src->dst} sent in the last round, for `slot`,
 * into dst_host (synchronises).  Before any round: zeros. */
int relaysum_get_message(relaysum_t *h, int32_t slot, float *dst_host);

/* Static name of a status code. */
const char *relaysum_strerror(int code);

/* Text of the last failure on this handle ("" if none); valid until the
 * next call on the handle. */
const char *relaysum_last_error(const relaysum_t *h);

#ifdef __cplusplus
}
#endif

#endif /* RELAYSUM_H */
