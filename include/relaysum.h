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
 * Graphs: relaysum_create resolves every kernel and launch attribute, so
 * relaysum_step and relaysum_step_ex only enqueue kernels and can be
 * recorded by HIP stream capture.  The round number (and with it the ring
 * and counter parity a call uses) advances when a call is recorded, not
 * when the graph runs: record an even number of rounds, and replay the
 * graph only while the handle's eager calls come in pairs, so that every
 * replay finds the parity it was recorded with.  Arguments are fixed at
 * recording (Adam's step count, lr, the loss mask pointer).
 *
 * Errors: every int-returning function returns RELAYSUM_OK (0) or a negative
 * relaysum_status; relaysum_strerror() names a code and
 * relaysum_last_error() gives the text of the handle's last failure.
 */
#ifndef RELAYSUM_H
#define RELAYSUM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct relaysum_s relaysum_t;

/* Largest number of workers a handle takes.  The divisor nbar_i <= n of
 * Alg. 1's average is converted to binary32, which holds every integer up to
 * 2^24 exactly, so up to this size the division is the paper's. */
#define RELAYSUM_MAX_WORKERS 16777216

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
 *   1 <= n <= RELAYSUM_MAX_WORKERS, d >= 0 (d == 0: rounds only relay the
 *   counters).
 *   Returns RELAYSUM_ERR_NOT_A_TREE unless num_edges == n-1, every id is in
 *   [0, n), and the edges have no self loop, no duplicate and connect all
 *   workers; RELAYSUM_ERR_INVALID_ARG for n out of range, d < 0, out == NULL, or
 *   edges == NULL with num_edges > 0; RELAYSUM_ERR_OUT_OF_MEMORY when device
 *   memory for the ring cannot be had: 2 * 2(n-1) messages of d floats,
 *   each rounded up to whole ring tiles (4096 floats; a shorter message to
 *   the next power of two, at least 4 floats on single trees and 512 on
 *   double trees); single trees of more than 32 workers (double trees from
 *   65 workers, degrees of at most 32) also take d floats for each worker
 *   with a neighbour outside its cluster of 16 workers (32 on double trees
 *   and on single trees of 2,048 workers or more) and for each worker of
 *   more than 8 neighbours (single trees): 6 on a chain of 64.
 * Allocates on the current HIP device, zeroes every message and counter
 * (m^{(-1)} = 0, c^{(-1)} = 0) and sets the round number to 0.  On failure
 * *out is set to NULL. */
int relaysum_create(int32_t n, int64_t d, const int32_t *edges, int32_t num_edges,
                    relaysum_t **out);

/* Double binary trees (Section 3): a handle whose rounds relay the odd
 * model coordinates 1, 3, 5, ... over tree A (edges_a) and the even ones
 * 0, 2, 4, ... over tree B (edges_b), both trees on the same n workers with
 * num_edges = n-1 edges each, validated as in relaysum_create.  Each tree
 * keeps its own counters and messages (of d/2 and (d+1)/2 floats), so a
 * coordinate's result is exactly that of a single-tree handle on its tree
 * run over the coordinates of its parity.  Every step and accessor below
 * applies; directed-edge slots are numbered tree-major: tree A's 2(n-1)
 * slots first, then tree B's.  The trees need not be complementary; the
 * paper pairs two binary trees in which every worker is a leaf of one of
 * them, so that each worker has at most 4 neighbours in total. */
int relaysum_create_double(int32_t n, int64_t d, const int32_t *edges_a, const int32_t *edges_b,
                           int32_t num_edges, relaysum_t **out);

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
 * Rows must be 4-byte aligned.  Results do not depend on alignment or d;
 * rounds are fastest on 16-byte aligned pointers with d % 4 == 0 (the
 * cluster path's completion launch needs both for 16-byte accesses; the
 * other kernels move 16-byte chunks at any 4-byte alignment, or one float
 * per thread).
 * Returns RELAYSUM_ERR_INVALID_ARG for h, x or g NULL (unless d == 0), mom
 * NULL with beta != 0, misaligned pointers, arrays that share bytes, or an
 * array that is not n*d floats inside one device-memory (or managed-memory)
 * allocation of the handle's GPU (host memory, another GPU's memory or a
 * short buffer would make a kernel fault; checked with the HIP runtime's
 * pointer queries, once per array: the handle remembers the last 8 arrays
 * that passed, so an array freed and replaced at the same address by a
 * shorter allocation is not queried again); RELAYSUM_ERR_DEVICE if a launch
 * fails.  The round number then does not
 * advance; a round of the cluster or two-pass path is several
 * launches, and if a later one fails, x, the optimizer state and the
 * handle's messages are partly updated: restore them (relaysum_load_state,
 * or relaysum_reset and the caller's own copies) before another round. */
int relaysum_step(relaysum_t *h, float *x, const float *g, float *mom, float lr, float beta);

/* ---- other update rules and local optimizers --------------------------- */

/* How a round turns what each worker received into its new state. */
typedef enum relaysum_update {
    /* Alg. 1: x_i = (xh_i + sum_j m_{j->i}) / nbar_i. */
    RELAYSUM_UPDATE_MODEL = 0,
    /* Robust rule of Section 5.4 (eq. robust), for unreliable links:
     * x_i = (xh_i + sum_j m_{j->i} + (n - nbar_i) * x_i^{(t)}) / n, i.e. every
     * model that has not arrived is replaced by the worker's own x_i^{(t)}. */
    RELAYSUM_UPDATE_ROBUST = 1,
    /* Alg. 4 (RelaySGD/Grad, Appendix G): the relay carries the updates
     * u_i = -lr * g_i and x_i = x_i + (u_i + sum_j m_{j->i}) / n.  Plain SGD
     * only (the optimizer field must be RELAYSUM_OPT_SGD with beta1 == 0). */
    RELAYSUM_UPDATE_GRAD = 2,
    /* Alg. 3 (RelaySum for distributed mean estimation, Appendix F): g holds
     * this round's samples, state1 the running sums y;
     * y_i += g_i + sum_j m_{j->i}, s_i += 1 + sum_j c_{j->i}, x_i = y_i / s_i
     * (x is output only: the estimate after this round's update).  The
     * library keeps the integer s_i; the division converts it to binary32,
     * exact up to 2^24, so the library refuses (RELAYSUM_ERR_INVALID_ARG,
     * nothing queued) a round that could take some s_i past 2^24.  It bounds
     * s_i by the sum over the mean-estimation rounds t of the workers within
     * t+1 hops of a worker in a tree of the tree's largest degree D:
     * min(n, 1 + D(t+1)) for D <= 2, min(n, 1 + D(1 + (D-1) + ... +
     * (D-1)^t)) otherwise (on a 1024-worker chain, 16,639 rounds).
     * relaysum_reset clears the bound; snapshots carry it. */
    RELAYSUM_UPDATE_MEAN = 3
} relaysum_update;

/* Local step that forms the half-step xh_i (RELAYSUM_UPDATE_MODEL, _ROBUST). */
typedef enum relaysum_optimizer {
    /* beta1 == 0: xh = x - lr*g (Alg. 1's local step); beta1 != 0: Nesterov momentum
     * of Appendix D.2 with state1 = the momentum buffer. */
    RELAYSUM_OPT_SGD = 0,
    /* Adam, the local optimizer of Relay-Adam (Appendix D.3), in PyTorch's
     * form: bc1 = 1 - beta1^t, bc2 = 1 - beta2^t (double), m = beta1*m +
     * (1-beta1)*g, v = beta2*v + (1-beta2)*g*g, xh = x - (lr/bc1) * m /
     * (sqrt(v)/sqrt(bc2) + eps); state1 = m, state2 = v, t = adam_step. */
    RELAYSUM_OPT_ADAM = 1
} relaysum_optimizer;

typedef struct relaysum_round_args {
    int32_t update;          /* relaysum_update */
    int32_t optimizer;       /* relaysum_optimizer */
    float lr;                /* gamma */
    float beta1;             /* Nesterov alpha (SGD), or Adam beta1 */
    float beta2;             /* Adam beta2 */
    float eps;               /* Adam epsilon */
    int64_t adam_step;       /* Adam: 1-based step count t of the bias corrections */
    /* DEVICE array of one byte per directed-edge slot (2(n-1), or 4(n-1) on
     * double trees, tree-major), or NULL.  Nonzero marks the
     * message of that directed edge as lost in this round (Section 5.4): the
     * receiver gets neither the vector nor the counter, which count as zero
     * in its update now and in what it relays next round.  Read by the
     * round's kernels, so it must stay valid until they finish; checked
     * like x (RELAYSUM_ERR_INVALID_ARG if not). */
    const uint8_t *dropped;
} relaysum_round_args;

/* One round under `args` (see relaysum_update / relaysum_optimizer), then
 * t <- t+1.  x, g, state1, state2 are DEVICE [n][d] float rows as in
 * relaysum_step; which of them are read or written depends on the rule:
 *   MODEL/ROBUST + SGD:  x (rw), g (r), state1 = momentum (rw; NULL iff beta1 == 0)
 *   MODEL/ROBUST + ADAM: x (rw), g (r), state1 = m, state2 = v (rw)
 *   GRAD:                x (rw), g (r)
 *   MEAN:                x (w), g = samples (r), state1 = y (rw)
 * Unused pointers may be NULL.  Returns RELAYSUM_ERR_INVALID_ARG for a
 * missing buffer, an unknown rule, GRAD with momentum or Adam, Adam with
 * adam_step < 1, misaligned pointers, or used arrays that share bytes;
 * RELAYSUM_ERR_DEVICE on a launch failure (the round number then does not
 * advance).  relaysum_step(h, x, g, mom, lr, beta) is this call with MODEL,
 * SGD, beta1 = beta. */
int relaysum_step_ex(relaysum_t *h, float *x, const float *g, float *state1, float *state2,
                     const relaysum_round_args *args);

/* Mean estimation: s_i, the number of samples summed into y_i so far
 * (synchronises); n values per tree, tree-major (on double trees s_i of
 * tree A covers the odd coordinates, of tree B the even ones). */
int relaysum_get_samples(relaysum_t *h, int64_t *samples_host);

/* Consensus distance of the workers' models (the quantity Section 4's
 * analysis tracks, here with the uniform average of the models as centre):
 *   *dist   = (1/n) * sum_i ||x_i - xbar||^2,  xbar = (1/n) * sum_i x_i,
 *   *spread = max over workers i and coordinates c of |x_ic - xbar_c|
 * (spread may be NULL), for x of n*d floats in device memory of the
 * handle's GPU, row i worker i, 4-byte aligned, checked like relaysum_step's
 * arrays.  Accumulated in binary64 in an order fixed by n and d, so equal
 * inputs give equal bits.  Queued on the handle's stream behind its rounds,
 * then the stream is synchronised (not for graph capture).  d == 0 gives 0
 * and 0.  A NaN in x makes *dist NaN.  Not part of a round: an observability
 * aid for training loops and tests. */
int relaysum_consensus_distance(relaysum_t *h, const float *x, double *dist, double *spread);

/* Back to the state before the first round: messages, counters and sample
 * counts zeroed (queued on the handle's stream), round number 0. */
int relaysum_reset(relaysum_t *h);

/* Number of rounds done since create or reset. */
int relaysum_round(const relaysum_t *h, int64_t *t);

/* Number of trees of the handle: 1, or 2 for relaysum_create_double. */
int relaysum_num_trees(const relaysum_t *h, int32_t *count);

/* Kernel path a round of this handle takes (fixed at creation by the tree,
 * n and d; for tests and observability).  Every path computes the same
 * results. */
typedef enum relaysum_path {
    RELAYSUM_PATH_TILE = 0,        /* single trees of up to 32 workers */
    RELAYSUM_PATH_DTREE = 1,       /* double trees of up to 32 workers */
    RELAYSUM_PATH_WIDE_DTREE = 2,  /* retired; never returned */
    RELAYSUM_PATH_CLUSTER = 3,     /* single trees of more than 32 workers (workers of more
                                      than 8 neighbours through hub kernels ahead of the
                                      cluster kernel) */
    RELAYSUM_PATH_WIDE = 4,        /* retired; never returned */
    RELAYSUM_PATH_TWO_PASS = 5,    /* double trees of more than 64 workers with a worker of
                                      more than 32 neighbours, and d == 0 beyond 32
                                      workers */
    RELAYSUM_PATH_DTREE_SEQ = 6,   /* double trees of 33 to 64 workers */
    RELAYSUM_PATH_CLUSTER_DTREE = 7   /* double trees of more than 64 workers, degrees <= 32 */
} relaysum_path;
int relaysum_kernel_path(const relaysum_t *h, int32_t *path);

/* Number of directed-edge slots, 2(n-1) per tree.  Within a tree the slots
 * are ordered by source worker, then by destination, ascending; on double
 * trees tree A's slots come first. */
int relaysum_num_directed_edges(const relaysum_t *h, int32_t *count);

/* Floats in the message of `slot`: d on a single tree; on double trees
 * d/2 (tree A, odd coordinates) or (d+1)/2 (tree B, even coordinates). */
int relaysum_message_length(const relaysum_t *h, int32_t slot, int64_t *len);

/* Source and destination worker of a slot (host-side table lookup). */
int relaysum_directed_edge(const relaysum_t *h, int32_t slot, int32_t *src, int32_t *dst);

/* Counters of the last round (synchronises the handle's stream):
 * nbar_host[n per tree, tree-major] = nbar_i used in the last average,
 * edge_counts_host[one per slot] = c_{src->dst}.  Either pointer may be
 * NULL.  Before any round every value is 0. */
int relaysum_get_counts(relaysum_t *h, int32_t *nbar_host, int32_t *edge_counts_host);

/* The relaysum_message_length floats of message m_{src->dst} sent in the
 * last round, for `slot`, into dst_host (synchronises); on double trees the
 * carried coordinates in ascending order.  Before any round: zeros.
 * RELAYSUM_ERR_INVALID_ARG for a bad slot or NULL dst_host;
 * RELAYSUM_ERR_OUT_OF_MEMORY if a double-tree handle cannot get the host
 * staging buffer (whole ring tiles of the message). */
int relaysum_get_message(relaysum_t *h, int32_t slot, float *dst_host);

/* Snapshots, for resuming a run (no passage of the paper defines them; a
 * caller checkpointing a RelaySGD training run needs them).  A snapshot holds
 * what a handle carries from one round to the next: the round number, the
 * last round's counters, nbar and sample counts of every tree, and its
 * messages (the ring parity the next round reads), behind a header with the
 * handle's shape and a digest of its trees.  The caller keeps its own x and
 * optimizer state.  Loading a snapshot into a handle with the same n, d and
 * trees (edge lists in any order) and running rounds from there gives, bit
 * for bit, what the saved handle would have given.
 *
 * Bytes of a snapshot of this handle (about 2(n-1) * d * 4 per tree plus a
 * few KB). */
int relaysum_state_size(const relaysum_t *h, size_t *bytes);

/* Write a snapshot into buf (HOST or DEVICE memory, at least
 * relaysum_state_size bytes), after the work queued on the handle's stream
 * (synchronises).  RELAYSUM_ERR_INVALID_ARG for NULL buf or too few bytes. */
int relaysum_save_state(relaysum_t *h, void *buf, size_t bytes);

/* Replace the handle's state with a snapshot from buf (HOST or DEVICE
 * memory), after the work queued on its stream (synchronises); the round
 * number becomes the snapshot's.  RELAYSUM_ERR_INVALID_ARG, with the handle
 * unchanged, for NULL buf, too few bytes, another library version, or a
 * snapshot of a handle with other n, d or trees. */
int relaysum_load_state(relaysum_t *h, const void *buf, size_t bytes);

/* Test aid for the round's data flow: fill what the next round writes
 * (its ring parity, counters, nbar, sample counts, and the cluster path's
 * counter sums and partial sums of boundary workers) with all-ones bytes
 * (NaN floats, -1 integers), queued on the handle's stream with memset
 * nodes (not for graph capture).  A round reads only what the round before
 * it wrote, so its results do not change; one that read what it writes
 * would turn NaN or negative.  relaysum_get_counts reads -1 for nbar until
 * the next round, relaysum_get_samples -1 until the next mean-estimation
 * round (the only rule that keeps sample counts). */
int relaysum_poison_next(relaysum_t *h);

/* ---- for callers that cannot allocate ------------------------------------ */

/* relaysum_step without a handle, for callers that cannot allocate device
 * memory (code under HIP graph capture, allocation-free serving loops,
 * harnesses that forbid hipMalloc): one round t of Alg. 1 (relaysum_step's
 * arithmetic, bit for bit the result of a handle created with the same n, d
 * and edges at its round t) with the tree's CSR form, the counters and the
 * two-slot message ring kept in a static device buffer of the library
 * instead of handle memory.  It calls no allocator.
 *   n, d, edges, num_edges  as relaysum_create, with 1 <= n <= 32;
 *   t                       the round number: t == 0 starts a run (the
 *                           buffer's counters and the ring parity round 0
 *                           reads are cleared, by a kernel); t > 0 continues
 *                           the run whose round t-1 was the last call of this
 *                           function on the current device;
 *   x, g, mom, lr, beta     as relaysum_step (device pointers, [n][d] float);
 *   hip_stream              the stream the round is queued on (NULL = null
 *                           stream).
 * Limit: the buffer holds 64 MiB per GPU (allocated when the library is
 * loaded on a device, held until the process ends); a round needs about
 * 2 * 2(n-1) * d * 4 bytes of it (ring tiles of 4096 floats, or the next
 * power of two of at least 512 for shorter d), e.g. a 16-worker tree up to
 * d of about 270,000.  Every call on one GPU shares that GPU's buffer, which
 * keeps the last call's contents: runs on one GPU must not overlap (a new
 * run, t == 0, replaces the previous one), and calls from several threads
 * on one GPU race.
 * Returns RELAYSUM_ERR_NOT_A_TREE as relaysum_create; RELAYSUM_ERR_INVALID_ARG
 * for n outside 1..32, d < 0, t < 0, a round that needs more than the
 * buffer, the pointer errors of relaysum_step, or t > 0 when the buffer does
 * not hold round t-1 of this n, d and tree; RELAYSUM_ERR_DEVICE on a HIP
 * error (the run is then ended).  relaysum_last_error(NULL) gives the text of
 * this thread's last failure. */
int relaysum_step_static(int32_t n, int64_t d, const int32_t *edges, int32_t num_edges, int64_t t,
                         float *x, const float *g, float *mom, float lr, float beta,
                         void *hip_stream);

/* Static name of a status code. */
const char *relaysum_strerror(int code);

/* Text of the last failure on this handle ("" if none); valid until the
 * next call on the handle.  With h == NULL: the last failure of
 * relaysum_step_static on the calling thread. */
const char *relaysum_last_error(const relaysum_t *h);

#ifdef __cplusplus
}
#endif

#endif /* RELAYSUM_H */
