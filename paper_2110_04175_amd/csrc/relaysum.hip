// RelaySum round on CDNA4 (gfx950): HIP kernels and the C ABI of relaysum.h.
//
// One launch performs one round of the paper's RelaySum mechanism for every
// worker of the tree: each worker forms what it puts into the relay (the
// half-step of Alg. 1 with SGD, the Nesterov step of Appendix D.2 or Adam of
// Appendix D.3; the update of Alg. 4; the sample of Alg. 3), relays
// messages and integer counters over the tree edges, and forms its new state
// (the count-corrected average of Alg. 1, the robust rule of Section 5.4,
// the update sum of Alg. 4, or the running mean of Alg. 3).  Messages lost
// on a link (Section 5.4) are written as zeros by the sender, which is what
// the receiver sees of them.
//
// The round streams every model, gradient, optimizer-state and message row
// once; it does a few flops per float, so it is bound by HBM bandwidth (no
// contraction, no MFMA).  Layout in HBM:
//   x, g, state         caller-owned float[n][d], row stride d
//   ring                float[2][ceil(d/4096)][2E][4096]: parity t&1
//                       receives the messages of round t while parity
//                       (t-1)&1 holds those of round t-1 (messages shorter
//                       than 4096 floats get the next power of two as ring
//                       tile, at least 4 floats on single trees and 512 on
//                       double trees).  The ring is
//                       tile-major: the 4096 coordinates [4096k, 4096k+4096)
//                       of all 2E messages are one contiguous block, so the
//                       messages the workgroups of eight neighbouring tiles
//                       stream are adjacent in HBM instead of 2E rows d
//                       floats apart (5.19 -> 5.47 TB/s in a probe of this
//                       access pattern on MI355X with 512-float ring tiles;
//                       4096 is 2-3% faster again)
//   counts              int32[2][2E] double-buffered like the ring, nbar[n];
//                       int64[2][n] sample counts for mean estimation
//   tree                CSR: row_ptr[n+1]; slots row_ptr[i]..row_ptr[i+1]-1
//                       are the directed edges i->col[s], col ascending;
//                       rev[s] is the slot of the reverse edge; src[s] = i
//
// Tile kernel (trees up to 32 workers).  A workgroup owns one tile: the same
// 64*U*C = 512 consecutive coordinates of every row (U = 2 chunks of 4 floats
// per lane, moved as 16-byte accesses on rows that are 4-byte aligned; when
// d % 4 != 0 the row's last floats are moved one by one).  Each wave
// owns whole workers (worker i belongs to wave i mod W).  Phase 1: a wave
// streams worker i's rows and the previous messages into i, forms i's
// payload (kept in registers), writes the optimizer state and the messages
// i->j to HBM and to an LDS tile [2E][64*U*C].  After a barrier, phase 2
// forms i's new state from the payload and the LDS copies of the new
// messages into i.  New messages are read back from LDS, never from HBM, so
// every HBM byte of the round is touched exactly once; the accesses are
// non-temporal, as nothing is reused within a round (a round whose whole
// working set fits in half the MALL uses cache-allocating accesses instead:
// the next round touches all of it again).  Every workgroup first
// relays the (few) integer counters into LDS itself, so no grid-wide
// synchronisation is needed; workgroup 0 also publishes them.
//
// Double binary trees (Section 3): a second handle kind carries the odd
// coordinates on tree A and the even ones on tree B, each tree with its own
// counters.  Messages hold only their tree's coordinates (d/2 or (d+1)/2
// floats) and both trees share one ring, float[2][ceil((d+1)/8192)][4E][4096]
// with tree A's 2E slots first in each ring tile, so the message block of
// neighbouring workgroups stays one contiguous region as on a single tree.
// The double-tree kernel (up to 32 workers) streams x, g and the state once
// and splits every float4 into the pairs of the two trees; inside a ring
// tile a lane's two pairs of a tree sit together so that they move as one
// 16-byte access.
//
// Double trees of 33 to 64 workers relay one tree after the other through
// one LDS message tile (the sequential double-tree kernel); larger double
// trees of bounded degree run as clusters shared by both trees.
//
// Cluster kernels (single trees of more than 32 workers): the tree is cut
// into clusters of at most 16 workers built from connected subtrees.  One
// workgroup per (tile, cluster), one worker per wave, does the tile
// kernel's work for its cluster, with the messages inside the cluster in
// LDS; a worker with a neighbour in another cluster leaves its partial sum
// (payload plus the messages from neighbours before its first one outside
// the cluster) in a scratch array, and a second launch completes it from the
// ring.  On trees of at most 256 workers and degree at most 3 every
// workgroup relays the counters itself, as in the tile kernel; on the others
// they come from one small launch before.  Workers of more than 8
// neighbours (hubs) join no cluster: hub kernels ahead of the cluster kernel
// form their payloads (into their scratch rows) and out-messages, their
// previous messages loaded once into registers, or streamed once past a
// block of sums held in registers, so every hub's reads are linear in its
// degree; members read a hub's message from the ring in its place in the
// sum, and the second launch completes the hubs.
//
// Two-pass path (double trees of more than 64 workers with a worker of more
// than 32 neighbours, once per tree, and rounds with d == 0): one small
// launch relays the counters; pass A forms the payloads and new messages of
// the workers of at most 8 neighbours, the hub kernels those of the others;
// pass B forms the new states from the new messages.  Pass A leaves the
// Alg. 1 half-step in x; rules that need the old model as well recompute
// their payload in pass B from the stored optimizer state, with the same
// operations.
//
// Arithmetic: one IEEE binary32 rounding per operation, contraction off, sums
// start from the payload and add neighbours in ascending id, divisions and
// square roots are correctly rounded.  Results do not depend on the access
// width, the tile or the grid.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "relaysum.h"
#include "tree_plan.hpp"

#pragma clang fp contract(off)

namespace {

constexpr int kWave = 64;
constexpr int kMaxWaves = 16;       // 1024-thread workgroups
constexpr int kMaxDegInRegs = 4;    // previous messages into a worker kept in VGPRs
constexpr int kMaxDegInRegs2 = 8;   // the same in pass A and the cluster kernels without the relay;
                                    // workers of more neighbours (hubs) take the hub kernels
constexpr int kHubDeg = 64;         // hubs of 9 to 64 neighbours take relaysum_pass_a_hub
constexpr int kHubClass[3] = {16, 32, 64};   // its degree classes; more neighbours: the blocked hub kernel
static_assert(kHubClass[0] > kMaxDegInRegs2 && kHubClass[2] == kHubDeg, "hub classes");
constexpr int kNumHubClasses = 4;
// Floats per message per ring tile: 4096 (16 KB), i.e. eight 512-coordinate
// kernel tiles share one ring tile.  On MI355X, sweeping 2^9..2^16 on the
// 16-worker chain (d = 9.75M and 110M) and the double binary trees gave the
// fastest rounds at 2^12 (2-3% faster than 2^9 and than 2^16).
constexpr int kRingShift = 12;
constexpr int kDTreeU = 2;          // float4 chunks per lane in the double-tree kernel
constexpr int kClusterLowDeg = 3;   // cluster trees of at most this degree: per-workgroup relay
constexpr int kClusterMaxDeg = 32;  // double trees whose degrees stay within this take the cluster kernels
constexpr int kClusterDegInRegs = 8;   // previous messages into a worker the cluster kernel keeps in VGPRs
// Single trees of at least this many workers (whose kernel does not relay
// the counters) run clusters of 32, two members per wave: half the boundary
// rows of clusters of 16.  On MI355X, same box, bit for bit the same
// results: random trees of 4,096 workers (d = 80,000) 2.41 -> 2.36 ms per
// round and of 8,192 (d = 40,000) 2.43 -> 2.37 ms; at 100 to 1,000 workers
// they were 0.5-2% slower (prufer256 1.77 -> 1.79-1.80 ms), and the
// 2,000-worker preferential-attachment tree measured the same.
constexpr int kClusterPairFrom = 2048;
// A cluster member has at most as many neighbours as its kernel keeps
// previous messages in registers: the hubs (workers of more than
// kMaxDegInRegs2 neighbours) join no cluster, and the trees whose kernel
// relays the counters have degrees of at most kClusterLowDeg.
static_assert(kClusterDegInRegs == kMaxDegInRegs2 && kClusterLowDeg <= kMaxDegInRegs,
              "cluster members must fit the registers of their kernel");
constexpr size_t kMallBytes = (size_t)256 << 20;   // MI355X Infinity Cache (MALL)

// Text of the last failure of relaysum_step_static on this thread (it has no
// handle to keep it in).
thread_local char g_static_err[256] = "";

// ---- update rules --------------------------------------------------------

enum Rule : int {
    kModelSgd = 0,       // Alg. 1, xh = x - lr*g
    kModelNesterov = 1,  // Alg. 1 with the momentum step of Appendix D.2
    kModelAdam = 2,      // Alg. 1 with Adam (Appendix D.3)
    kRobustSgd = 3,      // eq. robust (Section 5.4), local steps as above
    kRobustNesterov = 4,
    kRobustAdam = 5,
    kGrad = 6,           // Alg. 4: the relay carries u = -lr*g
    kMean = 7,           // Alg. 3: the relay carries samples
    kNumRules = 8
};

template <int R>
struct RuleOf {
    static constexpr bool robust = R == kRobustSgd || R == kRobustNesterov || R == kRobustAdam;
    static constexpr bool nesterov = R == kModelNesterov || R == kRobustNesterov;
    static constexpr bool adam = R == kModelAdam || R == kRobustAdam;
    static constexpr bool grad = R == kGrad;
    static constexpr bool mean = R == kMean;
    static constexpr bool model = !robust && !grad && !mean;
    static constexpr bool reads_x = !mean;                 // x^{(t)} is an input
    static constexpr bool keeps_x = robust || grad;        // x^{(t)} needed by the update
    static constexpr bool uses_s1 = nesterov || adam || mean;
    static constexpr bool uses_s2 = adam;
};

// ---- lane vectors ----------------------------------------------------------

// A lane's share of one row within a tile: U chunks of C floats (C = 4 for
// 16-byte accesses, C = 2 or 1 where a kernel moves narrower pieces).  Chunk u of lane l lies at float offset
// (u*64 + l)*C from the tile start, so every wave-wide access covers 64*C
// contiguous floats (1 KB when C = 4).
template <int U, int C>
struct lanev {
    float v[U][C];
};

typedef float f4_t __attribute__((ext_vector_type(4)));
typedef float f2_t __attribute__((ext_vector_type(2)));
// A 16-byte chunk of a row that is only known to be 4-byte aligned: rows
// start d floats apart, and the caller's arrays need only 4-byte alignment.
// gfx950 executes such a 16-byte access as one load or store (unaligned
// global accesses are enabled under ROCm), so the compiler emits a single
// dwordx4 access for it.
typedef float f4u_t __attribute__((ext_vector_type(4), aligned(4)));

// Every model, gradient, state and message row is touched once per round,
// so loads and stores are non-temporal (streamed past the caches), NT = true.
// A round whose whole working set fits in the 256 MB MALL touches every byte
// of it again in the next round; the tile kernel then uses cache-allocating
// accesses (NT = false) so that the next round finds it there.
template <int C, bool NT = true>
__device__ __forceinline__ void load_chunk(const float *p, float (&r)[C]) {
    if constexpr (C == 4) {
        const f4u_t *q = reinterpret_cast<const f4u_t *>(p);
        const f4u_t t = NT ? __builtin_nontemporal_load(q) : *q;
        r[0] = t.x; r[1] = t.y; r[2] = t.z; r[3] = t.w;
    } else if constexpr (C == 2) {
        const f2_t *q = reinterpret_cast<const f2_t *>(p);
        const f2_t t = NT ? __builtin_nontemporal_load(q) : *q;
        r[0] = t.x; r[1] = t.y;
    } else {
#pragma unroll
        for (int k = 0; k < C; ++k) r[k] = NT ? __builtin_nontemporal_load(p + k) : p[k];
    }
}

template <int C, bool NT = true>
__device__ __forceinline__ void store_chunk(float *p, const float (&a)[C]) {
    if constexpr (C == 4) {
        const f4u_t t = {a[0], a[1], a[2], a[3]};
        if constexpr (NT) __builtin_nontemporal_store(t, reinterpret_cast<f4u_t *>(p));
        else *reinterpret_cast<f4u_t *>(p) = t;
    } else if constexpr (C == 2) {
        const f2_t t = {a[0], a[1]};
        if constexpr (NT) __builtin_nontemporal_store(t, reinterpret_cast<f2_t *>(p));
        else *reinterpret_cast<f2_t *>(p) = t;
    } else {
#pragma unroll
        for (int k = 0; k < C; ++k) {
            if constexpr (NT) __builtin_nontemporal_store(a[k], p + k);
            else p[k] = a[k];
        }
    }
}

// Load a lane's chunks of one row; `row` points at the tile start of the row.
template <int U, int C, bool NT = true>
__device__ __forceinline__ lanev<U, C> load_lane(const float *row, int lane, const bool (&ok)[U]) {
    lanev<U, C> r;
#pragma unroll
    for (int u = 0; u < U; ++u) {
        if (ok[u]) {
            load_chunk<C, NT>(row + (u * 64 + lane) * C, r.v[u]);
        } else {
#pragma unroll
            for (int k = 0; k < C; ++k) r.v[u][k] = 0.0f;
        }
    }
    return r;
}

template <int U, int C, bool NT = true>
__device__ __forceinline__ void store_lane(float *row, int lane, const bool (&ok)[U],
                                           const lanev<U, C> &a) {
#pragma unroll
    for (int u = 0; u < U; ++u)
        if (ok[u]) store_chunk<C, NT>(row + (u * 64 + lane) * C, a.v[u]);
}

template <bool NT>
__device__ __forceinline__ float load_float(const float *p) {
    return NT ? __builtin_nontemporal_load(p) : *p;
}

template <bool NT>
__device__ __forceinline__ void store_float(float *p, float v) {
    if constexpr (NT) __builtin_nontemporal_store(v, p);
    else *p = v;
}

// The same with nv[u] valid floats in chunk u: C, or none past the row end,
// and with TAIL also fewer in the chunk holding the row's last coordinates
// when d % C != 0.  Whole chunks move as one access, the tail float by float.
// Without TAIL the code is that of the bool-mask form.
template <int U, int C, bool NT, bool TAIL>
__device__ __forceinline__ lanev<U, C> load_lane(const float *row, int lane, const int (&nv)[U]) {
    lanev<U, C> r;
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const float *p = row + (u * 64 + lane) * C;
        if (nv[u] == C) {
            load_chunk<C, NT>(p, r.v[u]);
        } else if constexpr (TAIL) {
#pragma unroll
            for (int k = 0; k < C; ++k) r.v[u][k] = k < nv[u] ? load_float<NT>(p + k) : 0.0f;
        } else {
#pragma unroll
            for (int k = 0; k < C; ++k) r.v[u][k] = 0.0f;
        }
    }
    return r;
}

template <int U, int C, bool NT, bool TAIL>
__device__ __forceinline__ void store_lane(float *row, int lane, const int (&nv)[U],
                                           const lanev<U, C> &a) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
        float *p = row + (u * 64 + lane) * C;
        if (nv[u] == C) {
            store_chunk<C, NT>(p, a.v[u]);
        } else if constexpr (TAIL) {
#pragma unroll
            for (int k = 0; k < C; ++k)
                if (k < nv[u]) store_float<NT>(p + k, a.v[u][k]);
        }
    }
}

template <int U, int C>
__device__ __forceinline__ lanev<U, C> zero_lane() {
    lanev<U, C> r;
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
        for (int k = 0; k < C; ++k) r.v[u][k] = 0.0f;
    return r;
}

template <int U, int C>
__device__ __forceinline__ lanev<U, C> add_lane(const lanev<U, C> &a, const lanev<U, C> &b) {
    lanev<U, C> r;
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
        for (int k = 0; k < C; ++k) r.v[u][k] = a.v[u][k] + b.v[u][k];
    return r;
}

// LDS copy of a lane's chunks: [slot][u][lane][C].
template <int U, int C>
__device__ __forceinline__ void lds_put(float *tile_slot, int lane, const lanev<U, C> &a) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
        float *p = tile_slot + (u * 64 + lane) * C;
        if constexpr (C == 4) {
            *reinterpret_cast<f4_t *>(p) = f4_t{a.v[u][0], a.v[u][1], a.v[u][2], a.v[u][3]};
        } else {
#pragma unroll
            for (int k = 0; k < C; ++k) p[k] = a.v[u][k];
        }
    }
}

template <int U, int C>
__device__ __forceinline__ lanev<U, C> lds_get(const float *tile_slot, int lane) {
    lanev<U, C> r;
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const float *p = tile_slot + (u * 64 + lane) * C;
        if constexpr (C == 4) {
            const f4_t t = *reinterpret_cast<const f4_t *>(p);
            r.v[u][0] = t.x; r.v[u][1] = t.y; r.v[u][2] = t.z; r.v[u][3] = t.w;
        } else {
#pragma unroll
            for (int k = 0; k < C; ++k) r.v[u][k] = p[k];
        }
    }
    return r;
}

// ---- kernel arguments ------------------------------------------------------

struct RoundArgs {
    float *x;
    const float *g;
    float *s1;                // Nesterov buffer, Adam m, or mean-estimation sums y
    float *s2;                // Adam v
    const float *ring_prev;   // messages of round t-1, [ring tiles][slots][2^ring_shift]
    float *ring_next;         // messages of round t
    int64_t d;                // floats per model row
    int64_t nchunks;          // d / C (C-float chunks per row)
    int64_t ntiles;           // tiles per row (64*U chunks each)
    const int32_t *cnt_prev;  // c^{(t-1)} per slot, as received
    int32_t *cnt_next;        // c^{(t)} per slot, as received
    int32_t *nbar_out;        // nbar_i of round t
    int32_t *cnt_sum;         // S_i: round t-1's counters into i, summed (cluster path with hubs)
    const int64_t *smp_prev;  // mean estimation: s_i before the round
    int64_t *smp_next;        // s_i after the round
    const uint8_t *dropped;   // lost messages of this round per slot, or nullptr
    const int32_t *row_ptr;
    const int32_t *col;
    const int32_t *rev;
    const int32_t *src;
    int32_t n;
    int32_t e2;
    int32_t ring_shift;       // log2 of the floats per message per ring tile
    int32_t ring_packed;      // double trees: lane-packed order inside a ring tile
    int32_t ring_slots;       // messages per ring tile (of every tree of the handle)
    int32_t cstride;          // two-pass path: model coordinate of carried coordinate j
    int32_t coff;             //   is coff + cstride * j (1, 0 for a single tree)
    float lr;
    float beta1;              // Nesterov alpha or Adam beta1
    float beta2;
    float eps;
    float one_m_b1;           // 1 - beta1 (binary32)
    float one_m_b2;           // 1 - beta2 (binary32)
    float step_size;          // Adam: lr / (1 - beta1^t), rounded once from double
    float bc2_sqrt;           // Adam: sqrt(1 - beta2^t), rounded once from double
    int64_t spill_base;       // tile kernel with a spill: first coordinate past the grid's tiles
    int32_t spill;            //   and the spill coordinates of each workgroup (at most 64)
    int32_t nhubs;            // workers of more than kMaxDegInRegs2 neighbours (hubs), by degree
    const int32_t *hubs;      //   class: the hub kernels take them, pass A and the clusters do not
    // Hub kernels ahead of the cluster kernel: ring positions of the slots
    // (nullptr: the slot itself), and the boundary scratch rows that receive
    // the hubs' payloads (nullptr: pass A's x), row hub_bidx[i] for hub i.
    const int32_t *hub_rpos;
    float *hub_pay;
    const int32_t *hub_bidx;
};

__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

// Position of carried coordinate w inside a lane-packed ring tile of a
// double-tree message: each 256-coordinate block belongs to one kernel tile,
// whose lane l holds the coordinate pairs 2l, 2l+1 and 128+2l, 128+2l+1 of
// the block and keeps all four in one 16-byte slot at 4l of the block.
__host__ __device__ __forceinline__ int64_t packed_pos(int64_t w) {
    return (w & ~(int64_t)255) | (((w >> 1) & 63) << 2) | (((w >> 7) & 1) << 1) | (w & 1);
}

// Address of message `slot` at carried coordinate c in a tile-major ring
// parity (ring tiles of 2^ring_shift floats; the two trees of a double-tree
// handle share the ring: a ring tile holds tree A's messages, then tree B's,
// and ring_prev/next of tree B point past tree A's slots).  Kernel tiles and
// chunks never straddle a ring tile.
__device__ __forceinline__ int64_t ring_off(const RoundArgs &a, int slot, int64_t c) {
    const int64_t rt = (int64_t)1 << a.ring_shift;
    const int64_t w = c & (rt - 1);
    return (((c >> a.ring_shift) * a.ring_slots + slot) << a.ring_shift) +
           (a.ring_packed ? packed_pos(w) : w);
}

// Topology read through the constant address space: with a wave-uniform
// index the load is a scalar one (scalar cache, counted apart from the row
// loads).  On MI355X the double-tree kernel (two trees' indices per worker)
// runs about 4% faster this way; the tile kernel keeps vector index loads,
// which measured 2-6% faster for it (their waits pace its ring loads behind
// its row loads).
__device__ __forceinline__ int ldc(const int32_t *p) {
    return *(const __attribute__((address_space(4))) int32_t *)p;
}

__device__ __forceinline__ bool lost(const RoundArgs &a, int slot) {
    return a.dropped != nullptr && a.dropped[slot] != 0;
}

// Counter relay (Alg. 1, 3) into LDS: c_{i->j} = 1 + sum_{k in N_i\j} c_{k->i}
// over the counters received last round (zero for a lost message), then
// nbar_i = 1 + sum_j c_{j->i}.  Mean estimation also sums s_i += nbar_i.
__device__ void relay_counts(const RoundArgs &a, int32_t *s_cnt, int32_t *s_nbar,
                             int64_t *s_smp) {
    for (int s = threadIdx.x; s < a.e2; s += blockDim.x) {
        const int i = a.src[s], j = a.col[s];
        int c = 1;
        for (int q = a.row_ptr[i]; q < a.row_ptr[i + 1]; ++q)
            if (a.col[q] != j) c += a.cnt_prev[a.rev[q]];
        s_cnt[s] = lost(a, s) ? 0 : c;
    }
    __syncthreads();
    for (int i = threadIdx.x; i < a.n; i += blockDim.x) {
        int nb = 1;
        for (int q = a.row_ptr[i]; q < a.row_ptr[i + 1]; ++q) nb += s_cnt[a.rev[q]];
        s_nbar[i] = nb;
        if (s_smp) s_smp[i] = a.smp_prev[i] + nb;
    }
    __syncthreads();
}

// relay_counts for the two trees of a double-tree round at once (one pair of
// barriers): threads take tree A's slots and workers, then tree B's.
__device__ void relay_counts2(const RoundArgs &a, const RoundArgs &b, int32_t *s_cnt_a,
                              int32_t *s_nbar_a, int64_t *s_smp_a, int32_t *s_cnt_b,
                              int32_t *s_nbar_b, int64_t *s_smp_b) {
    for (int k = threadIdx.x; k < a.e2 + b.e2; k += blockDim.x) {
        const bool in_a = k < a.e2;
        const RoundArgs &t = in_a ? a : b;
        const int s = in_a ? k : k - a.e2;
        const int i = t.src[s], j = t.col[s];
        int c = 1;
        for (int q = t.row_ptr[i]; q < t.row_ptr[i + 1]; ++q)
            if (t.col[q] != j) c += t.cnt_prev[t.rev[q]];
        (in_a ? s_cnt_a : s_cnt_b)[s] = lost(t, s) ? 0 : c;
    }
    __syncthreads();
    for (int k = threadIdx.x; k < 2 * a.n; k += blockDim.x) {
        const bool in_a = k < a.n;
        const RoundArgs &t = in_a ? a : b;
        const int i = in_a ? k : k - a.n;
        const int32_t *cnt = in_a ? s_cnt_a : s_cnt_b;
        int nb = 1;
        for (int q = t.row_ptr[i]; q < t.row_ptr[i + 1]; ++q) nb += cnt[t.rev[q]];
        (in_a ? s_nbar_a : s_nbar_b)[i] = nb;
        int64_t *smp = in_a ? s_smp_a : s_smp_b;
        if (smp) smp[i] = t.smp_prev[i] + nb;
    }
    __syncthreads();
}

__device__ void publish_counts(const RoundArgs &a, const int32_t *s_cnt, const int32_t *s_nbar,
                               const int64_t *s_smp) {
    for (int s = threadIdx.x; s < a.e2; s += blockDim.x) a.cnt_next[s] = s_cnt[s];
    for (int i = threadIdx.x; i < a.n; i += blockDim.x) {
        a.nbar_out[i] = s_nbar[i];
        if (s_smp) a.smp_next[i] = s_smp[i];
    }
}

// ---- the arithmetic of a round, per coordinate ------------------------------

// What worker i puts into the relay, one IEEE operation per line:
//   SGD (Alg. 1):              xh = x - lr*g
//   Nesterov (Appendix D.2):   b = beta*b + g; xh = x - lr*(g + beta*b)
//   Adam (Appendix D.3):       m = beta1*m + (1-beta1)*g; v = beta2*v + (1-beta2)*g*g;
//                              xh = x - (lr/bc1) * m / (sqrt(v)/sqrt(bc2) + eps)
//   Alg. 4:                    u = -(lr*g)
//   Alg. 3:                    the sample g
// s1, s2 hold the optimizer state on entry and its new value on exit.
template <int R, int U, int C>
__device__ __forceinline__ lanev<U, C> payload(const RoundArgs &a, const lanev<U, C> &x,
                                               const lanev<U, C> &g, lanev<U, C> &s1,
                                               lanev<U, C> &s2) {
    using T = RuleOf<R>;
    lanev<U, C> p;
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
        for (int k = 0; k < C; ++k) {
            const float gv = g.v[u][k];
            if constexpr (T::mean) {
                p.v[u][k] = gv;
            } else if constexpr (T::grad) {
                const float st = a.lr * gv;
                p.v[u][k] = -st;
            } else if constexpr (T::adam) {
                const float a1 = s1.v[u][k] * a.beta1;
                const float a2 = gv * a.one_m_b1;
                const float m = a1 + a2;
                const float q1 = s2.v[u][k] * a.beta2;
                const float gg = gv * gv;
                const float q2 = gg * a.one_m_b2;
                const float v = q1 + q2;
                s1.v[u][k] = m;
                s2.v[u][k] = v;
                const float r = __builtin_sqrtf(v);
                const float r2 = r / a.bc2_sqrt;
                const float den = r2 + a.eps;
                const float ratio = m / den;
                const float upd = a.step_size * ratio;
                p.v[u][k] = x.v[u][k] - upd;
            } else if constexpr (T::nesterov) {
                const float q0 = a.beta1 * s1.v[u][k];
                const float bn = q0 + gv;
                s1.v[u][k] = bn;
                const float q = a.beta1 * bn;
                const float w = gv + q;
                const float st = a.lr * w;
                p.v[u][k] = x.v[u][k] - st;
            } else {
                const float st = a.lr * gv;
                p.v[u][k] = x.v[u][k] - st;
            }
        }
    return p;
}

// Recompute the half-step from the optimizer state a payload() call has
// already updated (two-pass path, robust rules): the same operations.
template <int R, int C>
__device__ __forceinline__ lanev<1, C> half_step_again(const RoundArgs &a, const lanev<1, C> &x,
                                                       const lanev<1, C> &g, const lanev<1, C> &s1,
                                                       const lanev<1, C> &s2) {
    using T = RuleOf<R>;
    lanev<1, C> p;
#pragma unroll
    for (int k = 0; k < C; ++k) {
        if constexpr (T::adam) {
            const float r = __builtin_sqrtf(s2.v[0][k]);
            const float r2 = r / a.bc2_sqrt;
            const float den = r2 + a.eps;
            const float ratio = s1.v[0][k] / den;
            const float upd = a.step_size * ratio;
            p.v[0][k] = x.v[0][k] - upd;
        } else if constexpr (T::nesterov) {
            const float q = a.beta1 * s1.v[0][k];
            const float w = g.v[0][k] + q;
            const float st = a.lr * w;
            p.v[0][k] = x.v[0][k] - st;
        } else {
            const float st = a.lr * g.v[0][k];
            p.v[0][k] = x.v[0][k] - st;
        }
    }
    return p;
}

// New state of worker i from acc = payload + received messages (ascending):
//   Alg. 1:       x = acc / nbar
//   eq. robust:   x = (acc + (n - nbar) * x_old) / n
//   Alg. 4:       x = x_old + acc / n
//   Alg. 3:       y = y + acc; x = y / s
// For Alg. 3, `xo` carries y (in) and receives the new y (out).
template <int R, int U, int C>
__device__ __forceinline__ lanev<U, C> new_state(const RoundArgs &a, const lanev<U, C> &acc,
                                                 lanev<U, C> &xo, int nbar, int64_t smp) {
    using T = RuleOf<R>;
    lanev<U, C> xn;
    const float nb = (float)nbar;
    const float nf = (float)a.n;
    const float missing = (float)(a.n - nbar);
    const float sf = (float)smp;
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
        for (int k = 0; k < C; ++k) {
            if constexpr (T::robust) {
                const float w = missing * xo.v[u][k];
                const float tot = acc.v[u][k] + w;
                xn.v[u][k] = tot / nf;
            } else if constexpr (T::grad) {
                const float q = acc.v[u][k] / nf;
                xn.v[u][k] = xo.v[u][k] + q;
            } else if constexpr (T::mean) {
                const float y = xo.v[u][k] + acc.v[u][k];
                xo.v[u][k] = y;
                xn.v[u][k] = y / sf;
            } else {
                xn.v[u][k] = acc.v[u][k] / nb;
            }
        }
    return xn;
}

// Messages out of worker i (Alg. 1, 3, 4): for each neighbour j (slot
// s0+q), m_{i->j} = p_i + sum over the other in-edges b != q, ascending, of
// the previous round's m_{k->i}; a lost message is written as zeros.  `o`
// holds the previous messages when the degree is at most MD; larger degrees
// re-read them.  Each message goes to the ring and to the LDS tile.
template <int U, int C, int MD, bool NT, bool TAIL>
__device__ __forceinline__ void emit_messages(const RoundArgs &a, float *s_msg, int slot_floats,
                                              int lane, const int (&ok)[U], int64_t base, int s0,
                                              int deg, const lanev<U, C> &p,
                                              const lanev<U, C> (&o)[MD]) {
    if (deg <= MD) {
#pragma unroll
        for (int q = 0; q < MD; ++q) {
            if (q < deg) {
                lanev<U, C> m = p;
#pragma unroll
                for (int b = 0; b < MD; ++b)
                    if (b < deg && b != q) m = add_lane<U, C>(m, o[b]);
                if (lost(a, s0 + q)) m = zero_lane<U, C>();
                store_lane<U, C, NT, TAIL>(a.ring_next + ring_off(a, s0 + q, base), lane, ok, m);
                lds_put<U, C>(s_msg + (s0 + q) * slot_floats, lane, m);
            }
        }
    } else {
        for (int q = 0; q < deg; ++q) {
            lanev<U, C> m = p;
            for (int b = 0; b < deg; ++b) {
                if (b == q) continue;
                const int in_slot = uniform(a.rev[s0 + b]);
                m = add_lane<U, C>(
                    m, load_lane<U, C, NT, TAIL>(a.ring_prev + ring_off(a, in_slot, base), lane, ok));
            }
            if (lost(a, s0 + q)) m = zero_lane<U, C>();
            store_lane<U, C, NT, TAIL>(a.ring_next + ring_off(a, s0 + q, base), lane, ok, m);
            lds_put<U, C>(s_msg + (s0 + q) * slot_floats, lane, m);
        }
    }
}

// Tile of this workgroup.  Workgroups go to the eight XCDs round robin
// (workgroup b to XCD b mod 8), each XCD with its own L2.  Two consecutive
// tiles share a 128-byte line on every row whose start is not line-aligned
// (row i starts i*d*4 bytes into its array; on the 16-worker chain at
// d = 9.75M every odd row starts 64 bytes into a line), and on two XCDs that
// line is fetched from memory twice: 1.9% more reads than the round needs.
// Pairing tiles 2k and 2k+1 on one XCD (workgroups b and b+8 of each group
// of 16, dispatched close together) fetches it once.  On MI355X the
// single-tree tile kernel took 0.5-2% less time per round on that chain
// (FETCH_SIZE 3.101 -> 3.074 GB; eq. robust and Alg. 4 1-2% less, Alg. 3
// the same); groups of 4 or 8 tiles per XCD measured no gain.  The
// cache-allocating short rounds (3% slower paired), Adam (2-3% slower) and
// the double-tree kernels (1-4% slower, with their packed ring layout) keep
// the plain order.
template <bool PAIRED>
__device__ __forceinline__ int64_t tile_of_workgroup() {
    const int64_t b = blockIdx.x;
    if constexpr (!PAIRED) return b;
    const int64_t full = (int64_t)gridDim.x & ~(int64_t)15;
    return b < full ? 16 * (b >> 4) + 2 * (b & 7) + ((b >> 3) & 1) : b;
}

// ---- tile kernel -------------------------------------------------------------

// Workgroup b owns tile b, the 64*U*C consecutive coordinates starting at
// b*64*U*C, for every row.
//
// SP (spill): a grid of short rounds whose tiles exceed a whole number of
// dispatch rounds (of the workgroups that fit on the device at once) by a
// few would run its last tiles in one more dispatch round, at the cost of a
// whole tile's latency chain.  With SP the grid holds only the whole rounds'
// workgroups, and the coordinates past their tiles, [spill_base, d), are
// spread over the first of them: workgroup b also owns the a.spill (at most
// 64) coordinates from spill_base + b*spill that lie below d, one float per
// lane, with their own LDS message tile and their payloads parked in LDS
// across the main tile.  The spill goes first, so that its short latency
// chain precedes the main tile's instead of following it behind a second
// barrier; a workgroup whose spill is empty skips its memory accesses.
template <int U, int C, int PW, int R, bool NT, bool TAIL, bool SP>
__global__ void __launch_bounds__(1024) relaysum_tile_kernel(RoundArgs a) {
    using T = RuleOf<R>;
    extern __shared__ __align__(16) unsigned char smem[];
    int64_t *s_smp = reinterpret_cast<int64_t *>(smem);                 // [n] (mean only)
    int32_t *s_cnt = reinterpret_cast<int32_t *>(s_smp + (T::mean ? a.n : 0));
    int32_t *s_nbar = s_cnt + a.e2;
    const int hdr = (int)(((T::mean ? a.n * 8 : 0) + (a.e2 + a.n) * 4 + 15) & ~15);
    float *s_msg = reinterpret_cast<float *>(smem + hdr);               // [2E][U][64][C]
    constexpr int kSlot = 64 * U * C;                                    // floats per LDS slot

    relay_counts(a, s_cnt, s_nbar, T::mean ? s_smp : nullptr);
    if (blockIdx.x == 0) publish_counts(a, s_cnt, s_nbar, T::mean ? s_smp : nullptr);

    const int lane = threadIdx.x & (kWave - 1);
    const int wave = uniform(threadIdx.x >> 6);
    const int W = blockDim.x >> 6;
    const int64_t tile = tile_of_workgroup<NT && !T::adam>();
    const int64_t base = tile * kSlot;   // float offset of the tile in every row
    // Valid floats of each of this lane's chunks: C, 0 past the row end, and
    // with TAIL (d % C != 0) fewer in the chunk that holds the row's last
    // coordinates.
    int ok[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int64_t rem = a.d - (tile * 64 * U + u * 64 + lane) * C;
        ok[u] = rem >= C ? C : (TAIL && rem > 0 ? (int)rem : 0);
    }

    // Spill, phase 1: as phase 1 below, one float per lane; the payload (and
    // x^{(t)} or y where the update needs it) waits in LDS for phase 2.
    float *s_sp = s_msg + (size_t)a.e2 * kSlot;   // [2E][64] spill messages
    float *s_spay = s_sp + (size_t)a.e2 * kWave;  // [n][64] spill payloads
    float *s_sold = s_spay + (size_t)a.n * kWave; // [n][64] spill x^{(t)} or y
    int64_t sbase = 0;
    int oks[1] = {0};
    bool spilled = false;
    if constexpr (SP) {
        sbase = a.spill_base + (int64_t)blockIdx.x * a.spill;
        const int64_t send = sbase + a.spill < a.d ? sbase + a.spill : a.d;
        oks[0] = sbase + lane < send ? 1 : 0;
        spilled = sbase < a.d;
    }
    if (spilled) {
#pragma unroll
        for (int p = 0; p < PW; ++p) {
            const int i = wave + p * W;
            if (i >= a.n) break;
            const int64_t row = (int64_t)i * a.d + sbase;
            lanev<1, 1> xv = zero_lane<1, 1>(), s1 = zero_lane<1, 1>(), s2 = zero_lane<1, 1>();
            if constexpr (T::reads_x) xv = load_lane<1, 1, NT, false>(a.x + row, lane, oks);
            const lanev<1, 1> gv = load_lane<1, 1, NT, false>(a.g + row, lane, oks);
            if constexpr (T::uses_s1) s1 = load_lane<1, 1, NT, false>(a.s1 + row, lane, oks);
            if constexpr (T::uses_s2) s2 = load_lane<1, 1, NT, false>(a.s2 + row, lane, oks);
            const int s0 = uniform(a.row_ptr[i]);
            const int deg = uniform(a.row_ptr[i + 1]) - s0;
            lanev<1, 1> o[kMaxDegInRegs];
            if (deg <= kMaxDegInRegs) {
#pragma unroll
                for (int b = 0; b < kMaxDegInRegs; ++b) {
                    if (b < deg) {
                        const int in_slot = uniform(a.rev[s0 + b]);
                        o[b] = load_lane<1, 1, NT, false>(a.ring_prev + ring_off(a, in_slot, sbase),
                                                          lane, oks);
                    }
                }
            }
            const lanev<1, 1> pv = payload<R, 1, 1>(a, xv, gv, s1, s2);
            if constexpr (T::nesterov || T::adam) store_lane<1, 1, NT, false>(a.s1 + row, lane, oks, s1);
            if constexpr (T::adam) store_lane<1, 1, NT, false>(a.s2 + row, lane, oks, s2);
            emit_messages<1, 1, kMaxDegInRegs, NT, false>(a, s_sp, kWave, lane, oks, sbase, s0, deg,
                                                          pv, o);
            s_spay[i * kWave + lane] = pv.v[0][0];
            if constexpr (T::keeps_x) s_sold[i * kWave + lane] = xv.v[0][0];
            if constexpr (T::mean) s_sold[i * kWave + lane] = s1.v[0][0];
        }
    }

    lanev<U, C> pay[PW];   // payload of each owned worker
    lanev<U, C> old[PW];   // x^{(t)} (robust, Alg. 4) or y (Alg. 3)
    // Phase 1: payloads, optimizer state, outgoing messages.  All loads of a
    // worker are issued before any of its arithmetic.
#pragma unroll
    for (int p = 0; p < PW; ++p) {
        const int i = wave + p * W;
        if (i >= a.n) break;
        const int64_t row = (int64_t)i * a.d + base;
        lanev<U, C> xv = zero_lane<U, C>(), s1 = zero_lane<U, C>(), s2 = zero_lane<U, C>();
        if constexpr (T::reads_x) xv = load_lane<U, C, NT, TAIL>(a.x + row, lane, ok);
        const lanev<U, C> gv = load_lane<U, C, NT, TAIL>(a.g + row, lane, ok);
        if constexpr (T::uses_s1) s1 = load_lane<U, C, NT, TAIL>(a.s1 + row, lane, ok);
        if constexpr (T::uses_s2) s2 = load_lane<U, C, NT, TAIL>(a.s2 + row, lane, ok);
        const int s0 = uniform(a.row_ptr[i]);
        const int deg = uniform(a.row_ptr[i + 1]) - s0;
        lanev<U, C> o[kMaxDegInRegs];
        if (deg <= kMaxDegInRegs) {
#pragma unroll
            for (int b = 0; b < kMaxDegInRegs; ++b) {
                if (b < deg) {
                    const int in_slot = uniform(a.rev[s0 + b]);
                    o[b] = load_lane<U, C, NT, TAIL>(a.ring_prev + ring_off(a, in_slot, base), lane, ok);
                }
            }
        }
        pay[p] = payload<R, U, C>(a, xv, gv, s1, s2);
        if constexpr (T::keeps_x) old[p] = xv;
        if constexpr (T::mean) old[p] = s1;
        if constexpr (T::nesterov || T::adam) store_lane<U, C, NT, TAIL>(a.s1 + row, lane, ok, s1);
        if constexpr (T::adam) store_lane<U, C, NT, TAIL>(a.s2 + row, lane, ok, s2);
        emit_messages<U, C, kMaxDegInRegs, NT, TAIL>(a, s_msg, kSlot, lane, ok, base, s0, deg, pay[p], o);
    }
    __syncthreads();
    // Phase 2: new states.
#pragma unroll
    for (int p = 0; p < PW; ++p) {
        const int i = wave + p * W;
        if (i >= a.n) break;
        const int64_t row = (int64_t)i * a.d + base;
        const int s0 = uniform(a.row_ptr[i]);
        const int deg = uniform(a.row_ptr[i + 1]) - s0;
        lanev<U, C> acc = pay[p];
        for (int q = 0; q < deg; ++q) {
            const int in_slot = uniform(a.rev[s0 + q]);
            acc = add_lane<U, C>(acc, lds_get<U, C>(s_msg + in_slot * kSlot, lane));
        }
        lanev<U, C> xo = zero_lane<U, C>();
        if constexpr (T::keeps_x || T::mean) xo = old[p];
        const lanev<U, C> xn =
            new_state<R, U, C>(a, acc, xo, s_nbar[i], T::mean ? s_smp[i] : (int64_t)1);
        if constexpr (T::mean) store_lane<U, C, NT, TAIL>(a.s1 + row, lane, ok, xo);
        store_lane<U, C, NT, TAIL>(a.x + row, lane, ok, xn);
    }
    // Spill, phase 2.
    if (spilled) {
#pragma unroll
        for (int p = 0; p < PW; ++p) {
            const int i = wave + p * W;
            if (i >= a.n) break;
            const int64_t row = (int64_t)i * a.d + sbase;
            const int s0 = uniform(a.row_ptr[i]);
            const int deg = uniform(a.row_ptr[i + 1]) - s0;
            lanev<1, 1> acc;
            acc.v[0][0] = s_spay[i * kWave + lane];
            for (int q = 0; q < deg; ++q) {
                const int in_slot = uniform(a.rev[s0 + q]);
                acc = add_lane<1, 1>(acc, lds_get<1, 1>(s_sp + in_slot * kWave, lane));
            }
            lanev<1, 1> xo = zero_lane<1, 1>();
            if constexpr (T::keeps_x || T::mean) xo.v[0][0] = s_sold[i * kWave + lane];
            const lanev<1, 1> xn =
                new_state<R, 1, 1>(a, acc, xo, s_nbar[i], T::mean ? s_smp[i] : (int64_t)1);
            if constexpr (T::mean) store_lane<1, 1, NT, false>(a.s1 + row, lane, oks, xo);
            store_lane<1, 1, NT, false>(a.x + row, lane, oks, xn);
        }
    }
}

// ---- cluster kernels ------------------------------------------------------------

// Trees of more than 32 workers cut into clusters: connected subtrees of at most
// 16 workers (host: plan_clusters).  Workgroup b owns one 512-coordinate
// tile of one cluster: cluster b mod K of tile b / K, so the K clusters of a
// tile run on neighbouring workgroups.  Each wave owns one member.  Phase 1
// is the tile kernel's for the members: payload, optimizer state, every
// outgoing message to the ring, and the messages between members also to an
// LDS tile (slot k.lslot[s] of the cluster).  Phase 2 completes the members
// whose neighbours all lie in the cluster; a member with a neighbour in
// another cluster (a boundary worker) leaves in its row of the scratch array
// the canonical sum as far as the workgroup can take it (its payload plus
// the LDS messages of the neighbours before its first one in another
// cluster), and relaysum_cluster_fixup adds the remaining messages in a
// second launch, once every message of the round is in the ring.  No workgroup
// reads a row that another one writes in the same launch.  On trees of
// degree at most 3, as in the tile kernel, every workgroup relays the
// counters into LDS first (workgroup 0 publishes them), and long grids run
// one workgroup per CU: on MI355X the two together took chains of 64 and 256
// workers and a binary tree of 200 2-7% below a separate counter launch
// with two workgroups per CU.  On random trees (degrees 4 to 8) the relay in
// each of the many short workgroups costs far more (a chain of dependent
// loads over up to 510 counters), so relaysum_count_kernel writes the
// counters in a launch before and the grid runs uncapped.
struct ClusterArgs {
    const int32_t *members;   // [count][cap] worker ids, -1 past a cluster's size
    const int32_t *lslot;     // [2E]: LDS slot of a message inside its cluster, -1 across
    const int32_t *bidx;      // [n]: scratch row of a boundary worker, -1 otherwise
    const int32_t *bnd;       // [nb]: the boundary workers
    const int32_t *rpos;      // [2E]: ring position of a slot, each cluster's slots together
    const int32_t *bfirst;    // [nb]: index in N_i of a boundary worker's first neighbour in another cluster
    float *scratch;           // [nb][d]: their partial sums
    int32_t count;            // clusters K
    int32_t slots;            // LDS message slots of the largest cluster
    int32_t cap;              // 16 * PW
    int32_t nb;
};

// A cluster member's out-messages, from its payload and its previous
// in-messages in registers: a member has at most MD neighbours (a worker of
// more is a hub, which no cluster holds).
template <int U, int C, int MD, bool NT, bool TAIL>
__device__ __forceinline__ void emit_cluster_messages(const RoundArgs &a, const ClusterArgs &k,
                                                      float *s_msg, int lane, const int (&ok)[U],
                                                      int64_t base, int s0, int deg,
                                                      const lanev<U, C> &p,
                                                      const lanev<U, C> (&o)[MD]) {
    constexpr int kSlot = 64 * U * C;
#pragma unroll
    for (int q = 0; q < MD; ++q) {
        if (q < deg) {
            lanev<U, C> m = p;
#pragma unroll
            for (int b = 0; b < MD; ++b)
                if (b < deg && b != q) m = add_lane<U, C>(m, o[b]);
            if (lost(a, s0 + q)) m = zero_lane<U, C>();
            store_lane<U, C, NT, TAIL>(a.ring_next + ring_off(a, ldc(k.rpos + s0 + q), base), lane,
                                       ok, m);
            const int ls = ldc(k.lslot + s0 + q);
            if (ls >= 0) lds_put<U, C>(s_msg + ls * kSlot, lane, m);
        }
    }
}

// A round's message of slot `slot` into a cluster member, for its new
// state: from the cluster's LDS tile, or, with HUBS, from the ring for a
// message a hub kernel wrote before this launch (LDS slot -2).
template <int U, int C, bool NT, bool TAIL, bool HUBS>
__device__ __forceinline__ lanev<U, C> cluster_in_message(const RoundArgs &a, const ClusterArgs &k,
                                                          const float *s_msg, int lane,
                                                          const int (&ok)[U], int64_t base,
                                                          int slot) {
    constexpr int kSlot = 64 * U * C;
    const int ls = ldc(k.lslot + slot);
    if constexpr (HUBS) {
        if (ls < 0)
            return load_lane<U, C, NT, TAIL>(a.ring_next + ring_off(a, ldc(k.rpos + slot), base), lane, ok);
    }
    return lds_get<U, C>(s_msg + ls * kSlot, lane);
}

// MD: previous messages into a worker kept in VGPRs (a member has at most
// MD neighbours).  RELAY: counters relayed by every workgroup, as in the tile
// kernel, or by a launch before (nbar then read from memory); only the
// latter runs with hub kernels ahead of it, whose messages members read
// from the ring.
template <int U, int C, int MD, bool RELAY, int R, bool NT, bool TAIL, int PW>
__global__ void __launch_bounds__(1024) relaysum_cluster_kernel(RoundArgs a, ClusterArgs k) {
    using T = RuleOf<R>;
    extern __shared__ __align__(16) unsigned char smem[];
    int64_t *s_smp = reinterpret_cast<int64_t *>(smem);                 // [n] (mean only)
    int32_t *s_cnt = reinterpret_cast<int32_t *>(s_smp + (T::mean ? a.n : 0));
    int32_t *s_nbar = s_cnt + a.e2;
    const int hdr = RELAY ? (int)(((T::mean ? a.n * 8 : 0) + (a.e2 + a.n) * 4 + 15) & ~15) : 0;
    float *s_msg = reinterpret_cast<float *>(smem + hdr);               // [cluster slots][U][64][C]
    constexpr int kSlot = 64 * U * C;

    if constexpr (RELAY) {
        relay_counts(a, s_cnt, s_nbar, T::mean ? s_smp : nullptr);
        if (blockIdx.x == 0) publish_counts(a, s_cnt, s_nbar, T::mean ? s_smp : nullptr);
    }

    const int lane = threadIdx.x & (kWave - 1);
    const int wave = uniform(threadIdx.x >> 6);
    const int W = blockDim.x >> 6;
    const int cl = (int)(blockIdx.x % (unsigned)k.count);
    const int64_t tile = blockIdx.x / (unsigned)k.count;
    const int64_t base = tile * kSlot;
    const int32_t *mem = k.members + (int64_t)cl * k.cap;
    int ok[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int64_t rem = a.d - (tile * 64 * U + u * 64 + lane) * C;
        ok[u] = rem >= C ? C : (TAIL && rem > 0 ? (int)rem : 0);
    }

    lanev<U, C> pay[PW];
    lanev<U, C> old[PW];
#pragma unroll
    for (int p = 0; p < PW; ++p) {
        const int e = wave + p * W;
        const int i = e < k.cap ? ldc(mem + e) : -1;
        if (i < 0) break;
        const int64_t row = (int64_t)i * a.d + base;
        lanev<U, C> xv = zero_lane<U, C>(), s1 = zero_lane<U, C>(), s2 = zero_lane<U, C>();
        if constexpr (T::reads_x) xv = load_lane<U, C, NT, TAIL>(a.x + row, lane, ok);
        const lanev<U, C> gv = load_lane<U, C, NT, TAIL>(a.g + row, lane, ok);
        if constexpr (T::uses_s1) s1 = load_lane<U, C, NT, TAIL>(a.s1 + row, lane, ok);
        if constexpr (T::uses_s2) s2 = load_lane<U, C, NT, TAIL>(a.s2 + row, lane, ok);
        const int s0 = ldc(a.row_ptr + i);
        const int deg = ldc(a.row_ptr + i + 1) - s0;
        lanev<U, C> o[MD];
#pragma unroll
        for (int b = 0; b < MD; ++b) {
            if (b < deg) {
                const int in_pos = ldc(k.rpos + ldc(a.rev + s0 + b));
                o[b] = load_lane<U, C, NT, TAIL>(a.ring_prev + ring_off(a, in_pos, base), lane, ok);
            }
        }
        pay[p] = payload<R, U, C>(a, xv, gv, s1, s2);
        if constexpr (T::keeps_x) old[p] = xv;
        if constexpr (T::mean) old[p] = s1;
        if constexpr (T::nesterov || T::adam) store_lane<U, C, NT, TAIL>(a.s1 + row, lane, ok, s1);
        if constexpr (T::adam) store_lane<U, C, NT, TAIL>(a.s2 + row, lane, ok, s2);
        emit_cluster_messages<U, C, MD, NT, TAIL>(a, k, s_msg, lane, ok, base, s0, deg, pay[p], o);
    }
    __syncthreads();
#pragma unroll
    for (int p = 0; p < PW; ++p) {
        const int e = wave + p * W;
        const int i = e < k.cap ? ldc(mem + e) : -1;
        if (i < 0) break;
        const int s0 = ldc(a.row_ptr + i);
        const int deg = ldc(a.row_ptr + i + 1) - s0;
        const int b = ldc(k.bidx + i);
        if (b >= 0) {
            // Boundary worker: the canonical sum as far as this workgroup can
            // take it, up to its first neighbour in another cluster.
            const int qf = ldc(k.bfirst + b);
            lanev<U, C> part = pay[p];
            for (int q = 0; q < qf; ++q)
                part = add_lane<U, C>(part, cluster_in_message<U, C, NT, TAIL, !RELAY>(
                                                a, k, s_msg, lane, ok, base, ldc(a.rev + s0 + q)));
            store_lane<U, C, NT, TAIL>(k.scratch + (int64_t)b * a.d + base, lane, ok, part);
            continue;
        }
        const int64_t row = (int64_t)i * a.d + base;
        lanev<U, C> acc = pay[p];
        for (int q = 0; q < deg; ++q)
            acc = add_lane<U, C>(acc, cluster_in_message<U, C, NT, TAIL, !RELAY>(
                                          a, k, s_msg, lane, ok, base, ldc(a.rev + s0 + q)));
        lanev<U, C> xo = zero_lane<U, C>();
        if constexpr (T::keeps_x || T::mean) xo = old[p];
        int nbar;
        int64_t smp = 1;
        if constexpr (RELAY) {
            nbar = s_nbar[i];
            if constexpr (T::mean) smp = s_smp[i];
        } else {
            nbar = ldc(a.nbar_out + i);
            if constexpr (T::mean) smp = a.smp_next[i];
        }
        const lanev<U, C> xn = new_state<R, U, C>(a, acc, xo, nbar, smp);
        if constexpr (T::mean) store_lane<U, C, NT, TAIL>(a.s1 + row, lane, ok, xo);
        store_lane<U, C, NT, TAIL>(a.x + row, lane, ok, xn);
    }
}

// Boundary workers of a cluster round, boundary worker blockIdx.y
// (grid-strided): the partial sum the cluster kernel left in the scratch
// array (payload plus the messages from neighbours before the first one in
// another cluster) plus the round's remaining messages into them from the
// ring, ascending, then the new state.  Runs
// after relaysum_cluster_kernel, which has written every message, the
// counters and nbar; x^(t) (eq. robust, Alg. 4) and y (Alg. 3) of these
// workers are still unwritten.
template <int C, int R>
__global__ void __launch_bounds__(256) relaysum_cluster_fixup(RoundArgs a, ClusterArgs k) {
    using T = RuleOf<R>;
    const bool ok[1] = {true};
    for (int b = blockIdx.y; b < k.nb; b += gridDim.y) {
        const int i = k.bnd[b];
        const int s0 = a.row_ptr[i];
        const int deg = a.row_ptr[i + 1] - s0;
        const int nbar = a.nbar_out[i];
        const int64_t smp = T::mean ? a.smp_next[i] : (int64_t)1;
        for (int64_t chunk = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; chunk < a.nchunks;
             chunk += (int64_t)gridDim.x * blockDim.x) {
            const int64_t off = chunk * C;
            const int64_t row = (int64_t)i * a.d + off;
            lanev<1, C> xo = zero_lane<1, C>();
            if constexpr (T::keeps_x) xo = load_lane<1, C>(a.x + row, 0, ok);
            if constexpr (T::mean) xo = load_lane<1, C>(a.s1 + row, 0, ok);
            lanev<1, C> acc = load_lane<1, C>(k.scratch + (int64_t)b * a.d + off, 0, ok);
            // Eight messages loaded before they are added, in order: a hub's
            // completion walks hundreds of them.
            int q = k.bfirst[b];
            for (; q + 8 <= deg; q += 8) {
                lanev<1, C> m[8];
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    m[j] = load_lane<1, C>(a.ring_next + ring_off(a, k.rpos[a.rev[s0 + q + j]], off), 0, ok);
#pragma unroll
                for (int j = 0; j < 8; ++j) acc = add_lane<1, C>(acc, m[j]);
            }
            for (; q < deg; ++q)
                acc = add_lane<1, C>(
                    acc, load_lane<1, C>(a.ring_next + ring_off(a, k.rpos[a.rev[s0 + q]], off), 0, ok));
            const lanev<1, C> xn = new_state<R, 1, C>(a, acc, xo, nbar, smp);
            if constexpr (T::mean) store_lane<1, C>(a.s1 + row, 0, ok, xo);
            store_lane<1, C>(a.x + row, 0, ok, xn);
        }
    }
}

// ---- double binary trees ------------------------------------------------------

// A lane's two coordinate pairs of one tree (chunk u = 0, 1 of its float4s),
// moved as one 16-byte access: the ring and LDS tiles of a tree keep them
// together at float offset 4*lane (see packed_pos).
typedef lanev<kDTreeU, 2> pair2_t;
static_assert(kDTreeU == 2 && kRingShift >= 9,
              "packed_pos assumes 64 lanes x 2 chunks x 2 floats per 256-coordinate block");

__device__ __forceinline__ pair2_t load_pairs(const float *tile, int lane, bool ok) {
    pair2_t r;
    float t[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    if (ok) load_chunk<4>(tile + lane * 4, t);
    r.v[0][0] = t[0]; r.v[0][1] = t[1]; r.v[1][0] = t[2]; r.v[1][1] = t[3];
    return r;
}

__device__ __forceinline__ void store_pairs(float *tile, int lane, bool ok, const pair2_t &a) {
    const float t[4] = {a.v[0][0], a.v[0][1], a.v[1][0], a.v[1][1]};
    if (ok) store_chunk<4>(tile + lane * 4, t);
}

__device__ __forceinline__ void lds_put_pairs(float *slot, int lane, const pair2_t &a) {
    *reinterpret_cast<f4_t *>(slot + lane * 4) = f4_t{a.v[0][0], a.v[0][1], a.v[1][0], a.v[1][1]};
}

__device__ __forceinline__ pair2_t lds_get_pairs(const float *slot, int lane) {
    const f4_t t = *reinterpret_cast<const f4_t *>(slot + lane * 4);
    pair2_t r;
    r.v[0][0] = t.x; r.v[0][1] = t.y; r.v[1][0] = t.z; r.v[1][1] = t.w;
    return r;
}

// emit_messages for one tree of the double-tree kernel (packed tiles).
template <int MD>
__device__ __forceinline__ void emit_pair_messages(const RoundArgs &a, float *s_msg, int lane,
                                                   bool ok, int64_t tbase, int s0, int deg,
                                                   const pair2_t &p, const pair2_t (&o)[MD]) {
    constexpr int kSlot = 64 * kDTreeU * 2;
    if (deg <= MD) {
#pragma unroll
        for (int q = 0; q < MD; ++q) {
            if (q < deg) {
                pair2_t m = p;
#pragma unroll
                for (int b = 0; b < MD; ++b)
                    if (b < deg && b != q) m = add_lane<kDTreeU, 2>(m, o[b]);
                if (lost(a, s0 + q)) m = zero_lane<kDTreeU, 2>();
                store_pairs(a.ring_next + ring_off(a, s0 + q, tbase), lane, ok, m);
                lds_put_pairs(s_msg + (s0 + q) * kSlot, lane, m);
            }
        }
    } else {
        for (int q = 0; q < deg; ++q) {
            pair2_t m = p;
            for (int b = 0; b < deg; ++b) {
                if (b == q) continue;
                const int in_slot = ldc(a.rev + s0 + b);
                m = add_lane<kDTreeU, 2>(
                    m, load_pairs(a.ring_prev + ring_off(a, in_slot, tbase), lane, ok));
            }
            if (lost(a, s0 + q)) m = zero_lane<kDTreeU, 2>();
            store_pairs(a.ring_next + ring_off(a, s0 + q, tbase), lane, ok, m);
            lds_put_pairs(s_msg + (s0 + q) * kSlot, lane, m);
        }
    }
}

// Section 3's double binary trees: coordinate c travels on tree A when c is
// odd and on tree B when it is even.  `a` and `b` carry the same rows and
// scalars and each tree's own topology, counters and ring slots (a tree's
// message holds only its parity's coordinates).  The workgroup reads x, g
// and the optimizer state once: each
// lane's float4 chunk splits into the even pair (tree B) and the odd pair
// (tree A), and each pair is relayed on its own tree, with its own LDS tile.
// Chunks of 4 model coordinates start at multiples of 4 from the row start
// (16-byte accesses at any 4-byte alignment), so every chunk holds two
// coordinates of each tree and a workgroup's 512 model coordinates are one
// 256-coordinate block of each tree; with TAIL (d % 4 != 0) the row's last
// chunk is partial and moves float by float.  A lane's ring and LDS data of
// a tree is written when its first chunk holds any coordinate (chunk 1 lies
// 64 chunks further on): pairs past the tree's length carry values of
// missing coordinates, which no row ever receives; the ring holds whole ring
// tiles, so the 16-byte access stays in bounds on the ragged last tile.
template <int PW, int R, bool TAIL>
__global__ void __launch_bounds__(1024) relaysum_dtree_kernel(RoundArgs a, RoundArgs b) {
    using T = RuleOf<R>;
    constexpr int U = kDTreeU;
    constexpr int kSlot = 64 * U * 2;                 // floats per tree LDS slot
    extern __shared__ __align__(16) unsigned char smem[];
    int64_t *s_smp_a = reinterpret_cast<int64_t *>(smem);
    int64_t *s_smp_b = s_smp_a + a.n;
    int32_t *s_cnt_a = reinterpret_cast<int32_t *>(s_smp_b + a.n);
    int32_t *s_nbar_a = s_cnt_a + a.e2;
    int32_t *s_cnt_b = s_nbar_a + a.n;
    int32_t *s_nbar_b = s_cnt_b + b.e2;
    const int hdr = (int)((a.n * 16 + (a.e2 + b.e2 + 2 * a.n) * 4 + 15) & ~15);
    float *s_msg_a = reinterpret_cast<float *>(smem + hdr);   // [2E_A][64][4]
    float *s_msg_b = s_msg_a + (size_t)a.e2 * kSlot;           // [2E_B][64][4]

    relay_counts2(a, b, s_cnt_a, s_nbar_a, T::mean ? s_smp_a : nullptr, s_cnt_b, s_nbar_b,
                  T::mean ? s_smp_b : nullptr);
    if (blockIdx.x == 0) {
        publish_counts(a, s_cnt_a, s_nbar_a, T::mean ? s_smp_a : nullptr);
        publish_counts(b, s_cnt_b, s_nbar_b, T::mean ? s_smp_b : nullptr);
    }

    const int lane = threadIdx.x & (kWave - 1);
    const int wave = uniform(threadIdx.x >> 6);
    const int W = blockDim.x >> 6;
    const int64_t tile = blockIdx.x;
    const int64_t base = tile * (64 * U * 4);   // model coordinate of the tile
    const int64_t tbase = tile * kSlot;         // carried coordinate in each tree
    int ok[U];   // valid model coordinates in each of the lane's chunks
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int64_t rem = a.d - (tile * 64 * U + u * 64 + lane) * 4;
        ok[u] = rem >= 4 ? 4 : (TAIL && rem > 0 ? (int)rem : 0);
    }
    const bool ok_r = ok[0] > 0;

    pair2_t pa[PW], pb[PW];       // payload halves: odd (tree A), even (tree B)
    lanev<U, 4> old[PW];          // x^{(t)} (robust, Alg. 4) or y (Alg. 3)
#pragma unroll
    for (int p = 0; p < PW; ++p) {
        const int i = wave + p * W;
        if (i >= a.n) break;
        const int64_t row = (int64_t)i * a.d + base;
        lanev<U, 4> xv = zero_lane<U, 4>(), s1 = zero_lane<U, 4>(), s2 = zero_lane<U, 4>();
        if constexpr (T::reads_x) xv = load_lane<U, 4, true, TAIL>(a.x + row, lane, ok);
        const lanev<U, 4> gv = load_lane<U, 4, true, TAIL>(a.g + row, lane, ok);
        if constexpr (T::uses_s1) s1 = load_lane<U, 4, true, TAIL>(a.s1 + row, lane, ok);
        if constexpr (T::uses_s2) s2 = load_lane<U, 4, true, TAIL>(a.s2 + row, lane, ok);
        const int s0a = ldc(a.row_ptr + i), dega = ldc(a.row_ptr + i + 1) - s0a;
        const int s0b = ldc(b.row_ptr + i), degb = ldc(b.row_ptr + i + 1) - s0b;
        pair2_t oa[kMaxDegInRegs], ob[kMaxDegInRegs];
        if (dega <= kMaxDegInRegs) {
#pragma unroll
            for (int q = 0; q < kMaxDegInRegs; ++q)
                if (q < dega)
                    oa[q] = load_pairs(a.ring_prev + ring_off(a, ldc(a.rev + s0a + q), tbase), lane, ok_r);
        }
        if (degb <= kMaxDegInRegs) {
#pragma unroll
            for (int q = 0; q < kMaxDegInRegs; ++q)
                if (q < degb)
                    ob[q] = load_pairs(b.ring_prev + ring_off(b, ldc(b.rev + s0b + q), tbase), lane, ok_r);
        }
        const lanev<U, 4> pay = payload<R, U, 4>(a, xv, gv, s1, s2);
#pragma unroll
        for (int u = 0; u < U; ++u) {
            pb[p].v[u][0] = pay.v[u][0]; pb[p].v[u][1] = pay.v[u][2];
            pa[p].v[u][0] = pay.v[u][1]; pa[p].v[u][1] = pay.v[u][3];
        }
        if constexpr (T::keeps_x) old[p] = xv;
        if constexpr (T::mean) old[p] = s1;
        if constexpr (T::nesterov || T::adam) store_lane<U, 4, true, TAIL>(a.s1 + row, lane, ok, s1);
        if constexpr (T::adam) store_lane<U, 4, true, TAIL>(a.s2 + row, lane, ok, s2);
        emit_pair_messages<kMaxDegInRegs>(a, s_msg_a, lane, ok_r, tbase, s0a, dega, pa[p], oa);
        emit_pair_messages<kMaxDegInRegs>(b, s_msg_b, lane, ok_r, tbase, s0b, degb, pb[p], ob);
    }
    __syncthreads();
#pragma unroll
    for (int p = 0; p < PW; ++p) {
        const int i = wave + p * W;
        if (i >= a.n) break;
        const int64_t row = (int64_t)i * a.d + base;
        const int s0a = ldc(a.row_ptr + i), dega = ldc(a.row_ptr + i + 1) - s0a;
        const int s0b = ldc(b.row_ptr + i), degb = ldc(b.row_ptr + i + 1) - s0b;
        pair2_t acca = pa[p], accb = pb[p];
        for (int q = 0; q < dega; ++q)
            acca = add_lane<U, 2>(acca, lds_get_pairs(s_msg_a + ldc(a.rev + s0a + q) * kSlot, lane));
        for (int q = 0; q < degb; ++q)
            accb = add_lane<U, 2>(accb, lds_get_pairs(s_msg_b + ldc(b.rev + s0b + q) * kSlot, lane));
        pair2_t oa = zero_lane<U, 2>(), ob = zero_lane<U, 2>();
        if constexpr (T::keeps_x || T::mean) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                ob.v[u][0] = old[p].v[u][0]; ob.v[u][1] = old[p].v[u][2];
                oa.v[u][0] = old[p].v[u][1]; oa.v[u][1] = old[p].v[u][3];
            }
        }
        const pair2_t xa = new_state<R, U, 2>(a, acca, oa, s_nbar_a[i], T::mean ? s_smp_a[i] : (int64_t)1);
        const pair2_t xb = new_state<R, U, 2>(b, accb, ob, s_nbar_b[i], T::mean ? s_smp_b[i] : (int64_t)1);
        lanev<U, 4> xn, yn;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            xn.v[u][0] = xb.v[u][0]; xn.v[u][1] = xa.v[u][0];
            xn.v[u][2] = xb.v[u][1]; xn.v[u][3] = xa.v[u][1];
            yn.v[u][0] = ob.v[u][0]; yn.v[u][1] = oa.v[u][0];
            yn.v[u][2] = ob.v[u][1]; yn.v[u][3] = oa.v[u][1];
        }
        if constexpr (T::mean) store_lane<U, 4, true, TAIL>(a.s1 + row, lane, ok, yn);
        store_lane<U, 4, true, TAIL>(a.x + row, lane, ok, xn);
    }
}

// Double binary trees of 33 to 64 workers.  Both trees' message tiles of a
// 512-coordinate tile (2 x 126 slots of 1 KB at 64 workers) would not fit in
// LDS together, one would: the workgroup relays the trees one after the
// other through the same LDS tile.  Phase 1 reads every worker's x, g and
// optimizer state once (each wave owns PW workers), forms the payload, writes
// the optimizer state and relays tree A (the odd coordinates); phase 2 forms
// tree A's new states, which stay in registers; phase 3 relays tree B (the
// even coordinates) from the payloads kept in registers, through the same
// LDS tile; phase 4 forms tree B's new states and writes both, interleaved,
// in one store.  Every HBM byte of the round is touched once: no message is
// read back and no row is read twice.  Ring layout, chunks and TAIL variant
// are the double-tree kernel's.
template <int PW, int R, bool TAIL>
__global__ void __launch_bounds__(1024) relaysum_dtree_seq_kernel(RoundArgs a, RoundArgs b) {
    using T = RuleOf<R>;
    constexpr int U = kDTreeU;
    constexpr int kSlot = 64 * U * 2;                 // floats per tree LDS slot
    extern __shared__ __align__(16) unsigned char smem[];
    int64_t *s_smp_a = reinterpret_cast<int64_t *>(smem);
    int64_t *s_smp_b = s_smp_a + a.n;
    int32_t *s_cnt_a = reinterpret_cast<int32_t *>(s_smp_b + a.n);
    int32_t *s_nbar_a = s_cnt_a + a.e2;
    int32_t *s_cnt_b = s_nbar_a + a.n;
    int32_t *s_nbar_b = s_cnt_b + b.e2;
    const int hdr = (int)((a.n * 16 + (a.e2 + b.e2 + 2 * a.n) * 4 + 15) & ~15);
    float *s_msg = reinterpret_cast<float *>(smem + hdr);   // [max(2E_A, 2E_B)][64][4]

    relay_counts2(a, b, s_cnt_a, s_nbar_a, T::mean ? s_smp_a : nullptr, s_cnt_b, s_nbar_b,
                  T::mean ? s_smp_b : nullptr);
    if (blockIdx.x == 0) {
        publish_counts(a, s_cnt_a, s_nbar_a, T::mean ? s_smp_a : nullptr);
        publish_counts(b, s_cnt_b, s_nbar_b, T::mean ? s_smp_b : nullptr);
    }

    const int lane = threadIdx.x & (kWave - 1);
    const int wave = uniform(threadIdx.x >> 6);
    const int W = blockDim.x >> 6;
    const int64_t tile = blockIdx.x;
    const int64_t base = tile * (64 * U * 4);   // model coordinate of the tile
    const int64_t tbase = tile * kSlot;         // carried coordinate in each tree
    int ok[U];   // valid model coordinates in each of the lane's chunks
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int64_t rem = a.d - (tile * 64 * U + u * 64 + lane) * 4;
        ok[u] = rem >= 4 ? 4 : (TAIL && rem > 0 ? (int)rem : 0);
    }
    const bool ok_r = ok[0] > 0;

    pair2_t pa[PW], pb[PW];   // payload halves; pa becomes tree A's new state
    lanev<U, 4> old[PW];      // x^{(t)} (robust, Alg. 4) or y (Alg. 3); Alg. 3 keeps tree A's new y in it
    // Phase 1: rows, payloads, optimizer state, tree A's messages.
#pragma unroll
    for (int p = 0; p < PW; ++p) {
        const int i = wave + p * W;
        if (i >= a.n) break;
        const int64_t row = (int64_t)i * a.d + base;
        lanev<U, 4> xv = zero_lane<U, 4>(), s1 = zero_lane<U, 4>(), s2 = zero_lane<U, 4>();
        if constexpr (T::reads_x) xv = load_lane<U, 4, true, TAIL>(a.x + row, lane, ok);
        const lanev<U, 4> gv = load_lane<U, 4, true, TAIL>(a.g + row, lane, ok);
        if constexpr (T::uses_s1) s1 = load_lane<U, 4, true, TAIL>(a.s1 + row, lane, ok);
        if constexpr (T::uses_s2) s2 = load_lane<U, 4, true, TAIL>(a.s2 + row, lane, ok);
        const int s0a = ldc(a.row_ptr + i), dega = ldc(a.row_ptr + i + 1) - s0a;
        pair2_t oa[kMaxDegInRegs];
        if (dega <= kMaxDegInRegs) {
#pragma unroll
            for (int q = 0; q < kMaxDegInRegs; ++q)
                if (q < dega)
                    oa[q] = load_pairs(a.ring_prev + ring_off(a, ldc(a.rev + s0a + q), tbase), lane, ok_r);
        }
        const lanev<U, 4> pay = payload<R, U, 4>(a, xv, gv, s1, s2);
#pragma unroll
        for (int u = 0; u < U; ++u) {
            pb[p].v[u][0] = pay.v[u][0]; pb[p].v[u][1] = pay.v[u][2];
            pa[p].v[u][0] = pay.v[u][1]; pa[p].v[u][1] = pay.v[u][3];
        }
        if constexpr (T::keeps_x) old[p] = xv;
        if constexpr (T::mean) old[p] = s1;
        if constexpr (T::nesterov || T::adam) store_lane<U, 4, true, TAIL>(a.s1 + row, lane, ok, s1);
        if constexpr (T::adam) store_lane<U, 4, true, TAIL>(a.s2 + row, lane, ok, s2);
        emit_pair_messages<kMaxDegInRegs>(a, s_msg, lane, ok_r, tbase, s0a, dega, pa[p], oa);
    }
    __syncthreads();
    // Phase 2: tree A's new states (odd coordinates).
#pragma unroll
    for (int p = 0; p < PW; ++p) {
        const int i = wave + p * W;
        if (i >= a.n) break;
        const int s0a = ldc(a.row_ptr + i), dega = ldc(a.row_ptr + i + 1) - s0a;
        pair2_t acc = pa[p];
        for (int q = 0; q < dega; ++q)
            acc = add_lane<U, 2>(acc, lds_get_pairs(s_msg + ldc(a.rev + s0a + q) * kSlot, lane));
        pair2_t oa = zero_lane<U, 2>();
        if constexpr (T::keeps_x || T::mean) {
#pragma unroll
            for (int u = 0; u < U; ++u) { oa.v[u][0] = old[p].v[u][1]; oa.v[u][1] = old[p].v[u][3]; }
        }
        pa[p] = new_state<R, U, 2>(a, acc, oa, s_nbar_a[i], T::mean ? s_smp_a[i] : (int64_t)1);
        if constexpr (T::mean) {
#pragma unroll
            for (int u = 0; u < U; ++u) { old[p].v[u][1] = oa.v[u][0]; old[p].v[u][3] = oa.v[u][1]; }
        }
    }
    __syncthreads();   // the LDS tile is reused for tree B
    // Phase 3: tree B's messages.  The previous messages into all of the
    // wave's workers are loaded first (up to MB each, a binary tree's
    // degree; two for Alg. 3, which keeps y in registers as well), so that
    // one wait covers them: on MI355X 2-8% faster per round than loading
    // them worker by worker (48 and 64 workers).
    constexpr int MB = T::mean ? 2 : 3;
    pair2_t ob[PW][MB];
#pragma unroll
    for (int p = 0; p < PW; ++p) {
        const int i = wave + p * W;
        if (i < a.n) {
            const int s0b = ldc(b.row_ptr + i), degb = ldc(b.row_ptr + i + 1) - s0b;
            if (degb <= MB) {
#pragma unroll
                for (int q = 0; q < MB; ++q)
                    if (q < degb)
                        ob[p][q] = load_pairs(b.ring_prev + ring_off(b, ldc(b.rev + s0b + q), tbase), lane, ok_r);
            }
        }
    }
#pragma unroll
    for (int p = 0; p < PW; ++p) {
        const int i = wave + p * W;
        if (i >= a.n) break;
        const int s0b = ldc(b.row_ptr + i), degb = ldc(b.row_ptr + i + 1) - s0b;
        emit_pair_messages<MB>(b, s_msg, lane, ok_r, tbase, s0b, degb, pb[p], ob[p]);
    }
    __syncthreads();
    // Phase 4: tree B's new states (even coordinates); both trees' results
    // written interleaved.
#pragma unroll
    for (int p = 0; p < PW; ++p) {
        const int i = wave + p * W;
        if (i >= a.n) break;
        const int64_t row = (int64_t)i * a.d + base;
        const int s0b = ldc(b.row_ptr + i), degb = ldc(b.row_ptr + i + 1) - s0b;
        pair2_t acc = pb[p];
        for (int q = 0; q < degb; ++q)
            acc = add_lane<U, 2>(acc, lds_get_pairs(s_msg + ldc(b.rev + s0b + q) * kSlot, lane));
        pair2_t ob = zero_lane<U, 2>();
        if constexpr (T::keeps_x || T::mean) {
#pragma unroll
            for (int u = 0; u < U; ++u) { ob.v[u][0] = old[p].v[u][0]; ob.v[u][1] = old[p].v[u][2]; }
        }
        const pair2_t xb = new_state<R, U, 2>(b, acc, ob, s_nbar_b[i], T::mean ? s_smp_b[i] : (int64_t)1);
        const pair2_t &xa = pa[p];
        lanev<U, 4> xn, yn;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            xn.v[u][0] = xb.v[u][0]; xn.v[u][1] = xa.v[u][0];
            xn.v[u][2] = xb.v[u][1]; xn.v[u][3] = xa.v[u][1];
            yn.v[u][0] = ob.v[u][0]; yn.v[u][1] = old[p].v[u][1];
            yn.v[u][2] = ob.v[u][1]; yn.v[u][3] = old[p].v[u][3];
        }
        if constexpr (T::mean) store_lane<U, 4, true, TAIL>(a.s1 + row, lane, ok, yn);
        store_lane<U, 4, true, TAIL>(a.x + row, lane, ok, xn);
    }
}

// Double binary trees of more than 64 workers (both trees of degree at most
// kClusterMaxDeg), cut into clusters of at most 16 * PW workers shared by
// the two trees (host: plan_clusters_dual): the cluster kernel's scheme with
// the double-tree kernel's tiles, chunks and packed ring layout.  Workgroup
// b owns 512 model coordinates (256 of each tree) of one cluster, PW members
// per wave (wave, wave + 16, ...), whose payload pairs stay in registers
// across the barrier: phase 1 reads each member's rows once, forms the
// payload, splits it into the two trees' pairs and relays both trees (every message to the
// ring at the cluster layout's position, those between members also to the
// tree's LDS tile); phase 2 completes the members whose neighbours in both
// trees lie in the cluster, and leaves for a boundary worker (a neighbour in
// another cluster in either tree) both trees' canonical sums as far as the
// workgroup can take them, interleaved as a model row, in the scratch
// array; relaysum_cluster_dtree_fixup adds the remaining messages.  The
// counters come from relaysum_count_grid2_kernel, launched just before.
template <int MD>
__device__ __forceinline__ void emit_cluster_pairs(const RoundArgs &a, const ClusterArgs &k,
                                                   float *s_msg, int lane, bool ok, int64_t tbase,
                                                   int s0, int deg, const pair2_t &p,
                                                   const pair2_t (&o)[MD]) {
    constexpr int kSlot = 64 * kDTreeU * 2;
    if (deg <= MD) {
#pragma unroll
        for (int q = 0; q < MD; ++q) {
            if (q < deg) {
                pair2_t m = p;
#pragma unroll
                for (int c = 0; c < MD; ++c)
                    if (c < deg && c != q) m = add_lane<kDTreeU, 2>(m, o[c]);
                if (lost(a, s0 + q)) m = zero_lane<kDTreeU, 2>();
                store_pairs(a.ring_next + ring_off(a, ldc(k.rpos + s0 + q), tbase), lane, ok, m);
                const int ls = ldc(k.lslot + s0 + q);
                if (ls >= 0) lds_put_pairs(s_msg + ls * kSlot, lane, m);
            }
        }
    } else {
        for (int q = 0; q < deg; ++q) {
            pair2_t m = p;
            for (int c = 0; c < deg; ++c) {
                if (c == q) continue;
                const int in_pos = ldc(k.rpos + ldc(a.rev + s0 + c));
                m = add_lane<kDTreeU, 2>(m, load_pairs(a.ring_prev + ring_off(a, in_pos, tbase), lane, ok));
            }
            if (lost(a, s0 + q)) m = zero_lane<kDTreeU, 2>();
            store_pairs(a.ring_next + ring_off(a, ldc(k.rpos + s0 + q), tbase), lane, ok, m);
            const int ls = ldc(k.lslot + s0 + q);
            if (ls >= 0) lds_put_pairs(s_msg + ls * kSlot, lane, m);
        }
    }
}

template <int PW, int R, bool TAIL>
__global__ void __launch_bounds__(1024) relaysum_cluster_dtree_kernel(RoundArgs a, RoundArgs b,
                                                                      ClusterArgs ka, ClusterArgs kb) {
    using T = RuleOf<R>;
    constexpr int U = kDTreeU;
    constexpr int kSlot = 64 * U * 2;
    constexpr int MD = kMaxDegInRegs;
    extern __shared__ __align__(16) unsigned char smem[];
    float *s_msg_a = reinterpret_cast<float *>(smem);   // [slots of tree A][64][4]
    float *s_msg_b = s_msg_a + (size_t)ka.slots * kSlot;  // [slots of tree B][64][4]

    const int lane = threadIdx.x & (kWave - 1);
    const int wave = uniform(threadIdx.x >> 6);
    const int W = blockDim.x >> 6;
    const int cl = (int)(blockIdx.x % (unsigned)ka.count);
    const int64_t tile = blockIdx.x / (unsigned)ka.count;
    const int64_t base = tile * (64 * U * 4);
    const int64_t tbase = tile * kSlot;
    int ok[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int64_t rem = a.d - (tile * 64 * U + u * 64 + lane) * 4;
        ok[u] = rem >= 4 ? 4 : (TAIL && rem > 0 ? (int)rem : 0);
    }
    const bool ok_r = ok[0] > 0;

    int mem[PW];               // the wave's members: wave, wave + W, ... (-1 past the cluster)
    pair2_t pa[PW], pb[PW];
    lanev<U, 4> old[PW];
#pragma unroll
    for (int p = 0; p < PW; ++p) {
        const int e = wave + p * W;
        mem[p] = e < ka.cap ? ldc(ka.members + (int64_t)cl * ka.cap + e) : -1;
        old[p] = zero_lane<U, 4>();
    }
    // Phase 1, member by member: rows, payload, both trees' messages.
#pragma unroll
    for (int p = 0; p < PW; ++p) {
        const int i = mem[p];
        if (i < 0) continue;
        const int64_t row = (int64_t)i * a.d + base;
        lanev<U, 4> xv = zero_lane<U, 4>(), s1 = zero_lane<U, 4>(), s2 = zero_lane<U, 4>();
        if constexpr (T::reads_x) xv = load_lane<U, 4, true, TAIL>(a.x + row, lane, ok);
        const lanev<U, 4> gv = load_lane<U, 4, true, TAIL>(a.g + row, lane, ok);
        if constexpr (T::uses_s1) s1 = load_lane<U, 4, true, TAIL>(a.s1 + row, lane, ok);
        if constexpr (T::uses_s2) s2 = load_lane<U, 4, true, TAIL>(a.s2 + row, lane, ok);
        const int s0a = ldc(a.row_ptr + i), dega = ldc(a.row_ptr + i + 1) - s0a;
        const int s0b = ldc(b.row_ptr + i), degb = ldc(b.row_ptr + i + 1) - s0b;
        pair2_t oa[MD], ob[MD];
        if (dega <= MD) {
#pragma unroll
            for (int q = 0; q < MD; ++q)
                if (q < dega)
                    oa[q] = load_pairs(a.ring_prev + ring_off(a, ldc(ka.rpos + ldc(a.rev + s0a + q)), tbase),
                                       lane, ok_r);
        }
        if (degb <= MD) {
#pragma unroll
            for (int q = 0; q < MD; ++q)
                if (q < degb)
                    ob[q] = load_pairs(b.ring_prev + ring_off(b, ldc(kb.rpos + ldc(b.rev + s0b + q)), tbase),
                                       lane, ok_r);
        }
        const lanev<U, 4> pay = payload<R, U, 4>(a, xv, gv, s1, s2);
#pragma unroll
        for (int u = 0; u < U; ++u) {
            pb[p].v[u][0] = pay.v[u][0]; pb[p].v[u][1] = pay.v[u][2];
            pa[p].v[u][0] = pay.v[u][1]; pa[p].v[u][1] = pay.v[u][3];
        }
        if constexpr (T::keeps_x) old[p] = xv;
        if constexpr (T::mean) old[p] = s1;
        if constexpr (T::nesterov || T::adam) store_lane<U, 4, true, TAIL>(a.s1 + row, lane, ok, s1);
        if constexpr (T::adam) store_lane<U, 4, true, TAIL>(a.s2 + row, lane, ok, s2);
        emit_cluster_pairs<MD>(a, ka, s_msg_a, lane, ok_r, tbase, s0a, dega, pa[p], oa);
        emit_cluster_pairs<MD>(b, kb, s_msg_b, lane, ok_r, tbase, s0b, degb, pb[p], ob);
    }
    __syncthreads();
    // Phase 2.
#pragma unroll
    for (int p = 0; p < PW; ++p) {
        const int i = mem[p];
        if (i < 0) continue;
        const int s0a = ldc(a.row_ptr + i), dega = ldc(a.row_ptr + i + 1) - s0a;
        const int s0b = ldc(b.row_ptr + i), degb = ldc(b.row_ptr + i + 1) - s0b;
        const int bi = ldc(ka.bidx + i);
        // A boundary worker sums, in each tree, up to its first neighbour in
        // another cluster; every other worker all its neighbours.
        const int qa = bi >= 0 ? ldc(ka.bfirst + bi) : dega;
        const int qb = bi >= 0 ? ldc(kb.bfirst + bi) : degb;
        pair2_t acca = pa[p], accb = pb[p];
        for (int q = 0; q < qa; ++q)
            acca = add_lane<U, 2>(acca, lds_get_pairs(s_msg_a + ldc(ka.lslot + ldc(a.rev + s0a + q)) * kSlot, lane));
        for (int q = 0; q < qb; ++q)
            accb = add_lane<U, 2>(accb, lds_get_pairs(s_msg_b + ldc(kb.lslot + ldc(b.rev + s0b + q)) * kSlot, lane));
        if (bi >= 0) {
            lanev<U, 4> part;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                part.v[u][0] = accb.v[u][0]; part.v[u][1] = acca.v[u][0];
                part.v[u][2] = accb.v[u][1]; part.v[u][3] = acca.v[u][1];
            }
            store_lane<U, 4, true, TAIL>(ka.scratch + (int64_t)bi * a.d + base, lane, ok, part);
            continue;
        }
        pair2_t oa = zero_lane<U, 2>(), ob = zero_lane<U, 2>();
        if constexpr (T::keeps_x || T::mean) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                ob.v[u][0] = old[p].v[u][0]; ob.v[u][1] = old[p].v[u][2];
                oa.v[u][0] = old[p].v[u][1]; oa.v[u][1] = old[p].v[u][3];
            }
        }
        const pair2_t xa = new_state<R, U, 2>(a, acca, oa, ldc(a.nbar_out + i), T::mean ? a.smp_next[i] : (int64_t)1);
        const pair2_t xb = new_state<R, U, 2>(b, accb, ob, ldc(b.nbar_out + i), T::mean ? b.smp_next[i] : (int64_t)1);
        lanev<U, 4> xn, yn;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            xn.v[u][0] = xb.v[u][0]; xn.v[u][1] = xa.v[u][0];
            xn.v[u][2] = xb.v[u][1]; xn.v[u][3] = xa.v[u][1];
            yn.v[u][0] = ob.v[u][0]; yn.v[u][1] = oa.v[u][0];
            yn.v[u][2] = ob.v[u][1]; yn.v[u][3] = oa.v[u][1];
        }
        const int64_t row = (int64_t)i * a.d + base;
        if constexpr (T::mean) store_lane<U, 4, true, TAIL>(a.s1 + row, lane, ok, yn);
        store_lane<U, 4, true, TAIL>(a.x + row, lane, ok, xn);
    }
}

// Boundary workers of a double-tree cluster round, boundary worker
// blockIdx.y (grid-strided); each thread takes one lane of a 512-coordinate
// tile (the kernel's lanes, so the packed ring pieces are the kernel's): the
// partial sums from the scratch array plus, per tree, the round's messages
// from the first neighbour in another cluster on, then both new states.
template <int R, bool TAIL>
__global__ void __launch_bounds__(256) relaysum_cluster_dtree_fixup(RoundArgs a, RoundArgs b,
                                                                    ClusterArgs ka, ClusterArgs kb) {
    using T = RuleOf<R>;
    constexpr int U = kDTreeU;
    const int64_t lanes = a.ntiles * 64;
    for (int bi = blockIdx.y; bi < ka.nb; bi += gridDim.y) {
        const int i = ka.bnd[bi];
        const int s0a = a.row_ptr[i], dega = a.row_ptr[i + 1] - s0a;
        const int s0b = b.row_ptr[i], degb = b.row_ptr[i + 1] - s0b;
        const int qa = ka.bfirst[bi], qb = kb.bfirst[bi];
        const int nbar_a = a.nbar_out[i], nbar_b = b.nbar_out[i];
        const int64_t smp_a = T::mean ? a.smp_next[i] : (int64_t)1;
        const int64_t smp_b = T::mean ? b.smp_next[i] : (int64_t)1;
        for (int64_t gl = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; gl < lanes;
             gl += (int64_t)gridDim.x * blockDim.x) {
            const int64_t tile = gl >> 6;
            const int lane = (int)(gl & 63);
            const int64_t base = tile * (64 * U * 4);
            const int64_t tbase = tile * (64 * U * 2);
            int ok[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t rem = a.d - (tile * 64 * U + u * 64 + lane) * 4;
                ok[u] = rem >= 4 ? 4 : (TAIL && rem > 0 ? (int)rem : 0);
            }
            const bool ok_r = ok[0] > 0;
            const int64_t row = (int64_t)i * a.d + base;
            const lanev<U, 4> part = load_lane<U, 4, true, TAIL>(ka.scratch + (int64_t)bi * a.d + base, lane, ok);
            pair2_t acca, accb;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                accb.v[u][0] = part.v[u][0]; accb.v[u][1] = part.v[u][2];
                acca.v[u][0] = part.v[u][1]; acca.v[u][1] = part.v[u][3];
            }
            for (int q = qa; q < dega; ++q)
                acca = add_lane<U, 2>(acca, load_pairs(a.ring_next + ring_off(a, ka.rpos[a.rev[s0a + q]], tbase),
                                                       lane, ok_r));
            for (int q = qb; q < degb; ++q)
                accb = add_lane<U, 2>(accb, load_pairs(b.ring_next + ring_off(b, kb.rpos[b.rev[s0b + q]], tbase),
                                                       lane, ok_r));
            lanev<U, 4> old = zero_lane<U, 4>();
            if constexpr (T::keeps_x) old = load_lane<U, 4, true, TAIL>(a.x + row, lane, ok);
            if constexpr (T::mean) old = load_lane<U, 4, true, TAIL>(a.s1 + row, lane, ok);
            pair2_t oa = zero_lane<U, 2>(), ob = zero_lane<U, 2>();
            if constexpr (T::keeps_x || T::mean) {
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    ob.v[u][0] = old.v[u][0]; ob.v[u][1] = old.v[u][2];
                    oa.v[u][0] = old.v[u][1]; oa.v[u][1] = old.v[u][3];
                }
            }
            const pair2_t xa = new_state<R, U, 2>(a, acca, oa, nbar_a, smp_a);
            const pair2_t xb = new_state<R, U, 2>(b, accb, ob, nbar_b, smp_b);
            lanev<U, 4> xn, yn;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                xn.v[u][0] = xb.v[u][0]; xn.v[u][1] = xa.v[u][0];
                xn.v[u][2] = xb.v[u][1]; xn.v[u][3] = xa.v[u][1];
                yn.v[u][0] = ob.v[u][0]; yn.v[u][1] = oa.v[u][0];
                yn.v[u][2] = ob.v[u][1]; yn.v[u][3] = oa.v[u][1];
            }
            if constexpr (T::mean) store_lane<U, 4, true, TAIL>(a.s1 + row, lane, ok, yn);
            store_lane<U, 4, true, TAIL>(a.x + row, lane, ok, xn);
        }
    }
}

// ---- two-pass path --------------------------------------------------------

// Counter relay of the two-pass path (Alg. 1, 3), straight in global memory
// so that a tree of any size and degree fits, in one workgroup and O(2E)
// loads: with S_i = sum over all in-edges k -> i of c_{k->i}^{(t-1)} (kept in
// nbar_out meanwhile), c_{i->j}^{(t)} = 1 + S_i - c_{j->i}^{(t-1)}, exact in
// integers (every sum is at most n - 1, the workers on one side of i), or 0
// for a lost message; then, after the barrier that makes those writes
// visible to the workgroup, nbar_i = 1 + sum_j c_{j->i}^{(t)} and the sample
// counts.
__global__ void __launch_bounds__(1024) relaysum_count_kernel(RoundArgs a, int with_samples) {
    for (int i = threadIdx.x; i < a.n; i += blockDim.x) {
        int sum = 0;
        for (int q = a.row_ptr[i]; q < a.row_ptr[i + 1]; ++q) sum += a.cnt_prev[a.rev[q]];
        a.nbar_out[i] = sum;
    }
    __syncthreads();
    for (int s = threadIdx.x; s < a.e2; s += blockDim.x)
        a.cnt_next[s] = lost(a, s) ? 0 : 1 + a.nbar_out[a.src[s]] - a.cnt_prev[a.rev[s]];
    __syncthreads();
    for (int i = threadIdx.x; i < a.n; i += blockDim.x) {
        int nb = 1;
        for (int q = a.row_ptr[i]; q < a.row_ptr[i + 1]; ++q) nb += a.cnt_next[a.rev[q]];
        a.nbar_out[i] = nb;
        if (with_samples) a.smp_next[i] = a.smp_prev[i] + nb;
    }
}

// The same relay over many workgroups, for the cluster paths: thread k
// takes slot k (k < 2E) or worker
// k - 2E, and every value comes from round t-1's counters alone, so no
// thread waits for another's:
//   c_{i->j}^{(t)} = 1 + S_i - c_{j->i}^{(t-1)}             (0 if lost)
//   nbar_i         = 1 + sum_{j in N_i} c_{j->i}^{(t)},  with c_{j->i}^{(t)}
//                    = 1 + S_j - c_{i->j}^{(t-1)}            (0 if lost)
// where S_i sums the previous counters into i; a worker's nbar costs the sum
// of its neighbours' degrees in loads.
__device__ __forceinline__ int in_count_sum(const RoundArgs &a, int i) {
    int sum = 0;
    for (int q = a.row_ptr[i]; q < a.row_ptr[i + 1]; ++q) sum += a.cnt_prev[a.rev[q]];
    return sum;
}

// SUMS: S_i from a.cnt_sum, which a launch before filled, instead of
// summed here (a worker's nbar then costs its own degree in loads).
template <bool SUMS>
__device__ __forceinline__ int count_sum(const RoundArgs &a, int i) {
    return SUMS ? a.cnt_sum[i] : in_count_sum(a, i);
}

template <bool SUMS>
__device__ __forceinline__ void count_item(const RoundArgs &a, int k, int with_samples) {
    if (k < a.e2) {
        a.cnt_next[k] = lost(a, k) ? 0 : 1 + count_sum<SUMS>(a, a.src[k]) - a.cnt_prev[a.rev[k]];
    } else if (k < a.e2 + a.n) {
        const int i = k - a.e2;
        int nb = 1;
        for (int q = a.row_ptr[i]; q < a.row_ptr[i + 1]; ++q)
            if (!lost(a, a.rev[q])) nb += 1 + count_sum<SUMS>(a, a.col[q]) - a.cnt_prev[q];
        a.nbar_out[i] = nb;
        if (with_samples) a.smp_next[i] = a.smp_prev[i] + nb;
    }
}

template <bool SUMS>
__global__ void __launch_bounds__(256) relaysum_count_grid_kernel(RoundArgs a, int with_samples) {
    count_item<SUMS>(a, (int)(blockIdx.x * blockDim.x + threadIdx.x), with_samples);
}

// S_i for every worker i, one thread each, ahead of
// relaysum_count_grid_kernel<true>: on trees with hubs the sums over a
// worker's neighbours' in-counters would otherwise cost the workers next to
// hubs, and the hubs next to hubs, hundreds of loads in one thread (the
// 2,000-worker preferential-attachment tree: 57 us in one launch).
__global__ void __launch_bounds__(256) relaysum_count_sums_kernel(RoundArgs a) {
    const int i = (int)(blockIdx.x * blockDim.x + threadIdx.x);
    if (i < a.n) a.cnt_sum[i] = in_count_sum(a, i);
}

// Both trees of a double-tree round in one launch: tree A's items, then B's.
__global__ void __launch_bounds__(256) relaysum_count_grid2_kernel(RoundArgs a, RoundArgs b,
                                                                   int with_samples) {
    const int k = (int)(blockIdx.x * blockDim.x + threadIdx.x);
    const int na = a.e2 + a.n;
    if (k < na) count_item<false>(a, k, with_samples);
    else count_item<false>(b, k - na, with_samples);
}

// Pass A, worker blockIdx.y (grid-strided), for the workers of at most
// kMaxDegInRegs2 neighbours (the hub kernels take the others): payload,
// optimizer state and outgoing messages, the previous messages into i held
// in registers; for Alg. 1 the half-step is left in x for pass B.
template <int C, int R>
__global__ void __launch_bounds__(256) relaysum_pass_a(RoundArgs a) {
    using T = RuleOf<R>;
    const bool ok[1] = {true};
    constexpr int MD = kMaxDegInRegs2;
    for (int i = blockIdx.y; i < a.n; i += gridDim.y) {
        const int s0 = a.row_ptr[i];
        const int deg = a.row_ptr[i + 1] - s0;
        if (deg > MD) continue;   // a hub kernel's
        for (int64_t chunk = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; chunk < a.nchunks;
             chunk += (int64_t)gridDim.x * blockDim.x) {
            const int64_t off = chunk * C;
            const int64_t row = (int64_t)i * a.d + a.coff + a.cstride * off;
            lanev<1, C> xv = zero_lane<1, C>(), s1 = zero_lane<1, C>(), s2 = zero_lane<1, C>();
            if constexpr (T::reads_x) xv = load_lane<1, C>(a.x + row, 0, ok);
            const lanev<1, C> gv = load_lane<1, C>(a.g + row, 0, ok);
            if constexpr (T::nesterov || T::adam) s1 = load_lane<1, C>(a.s1 + row, 0, ok);
            if constexpr (T::adam) s2 = load_lane<1, C>(a.s2 + row, 0, ok);
            lanev<1, C> o[MD];
#pragma unroll
            for (int b = 0; b < MD; ++b)
                if (b < deg)
                    o[b] = load_lane<1, C>(a.ring_prev + ring_off(a, a.rev[s0 + b], off), 0, ok);
            const lanev<1, C> p = payload<R, 1, C>(a, xv, gv, s1, s2);
            if constexpr (T::nesterov || T::adam) store_lane<1, C>(a.s1 + row, 0, ok, s1);
            if constexpr (T::adam) store_lane<1, C>(a.s2 + row, 0, ok, s2);
            for (int q = 0; q < deg; ++q) {
                lanev<1, C> m = p;
#pragma unroll
                for (int b = 0; b < MD; ++b)
                    if (b < deg && b != q) m = add_lane<1, C>(m, o[b]);
                if (lost(a, s0 + q)) m = zero_lane<1, C>();
                store_lane<1, C>(a.ring_next + ring_off(a, s0 + q, off), 0, ok, m);
            }
            if constexpr (T::model) store_lane<1, C>(a.x + row, 0, ok, p);
        }
    }
}

// Ring position of slot s for the hub kernels: the slot itself on the
// two-pass path, the cluster plan's position ahead of the cluster kernel.
__device__ __forceinline__ int hub_pos(const RoundArgs &a, int s) {
    return a.hub_rpos ? ldc(a.hub_rpos + s) : s;
}

// Where a hub kernel leaves worker i's payload: x (pass B's input, Alg. 1
// only; the other rules recompute it there) on the two-pass path, or the
// worker's boundary scratch row, the start of the sum the cluster
// completion finishes, ahead of the cluster kernel (every rule; x^(t) stays
// in x for the rules that need it).
template <typename T>
__device__ __forceinline__ void store_hub_payload(const RoundArgs &a, int i, int64_t row, int64_t c,
                                                  const lanev<1, 1> &p) {
    const bool ok[1] = {true};
    if (a.hub_pay) store_lane<1, 1>(a.hub_pay + (int64_t)ldc(a.hub_bidx + i) * a.d + c, 0, ok, p);
    else if constexpr (T::model) store_lane<1, 1>(a.x + row, 0, ok, p);
}

// Pass A for the workers of kMaxDegInRegs2 + 1 to kHubDeg neighbours, in
// lists by degree class (at most DMAX = 16, 32 or 64 neighbours; a.hubs and
// a.nhubs name one class's list), hub h in blockIdx.y (grid-strided): one
// carried coordinate per thread, the worker's previous messages loaded once
// into registers, and every out-message summed from them in pass A's order
// (the payload, then the other in-messages ascending).  Each previous
// message is read once instead of once per out-message, so such a worker
// costs reads linear in its degree, not quadratic.  The registers past the
// degree hold -0.0, which leaves every IEEE sum unchanged (x + -0.0 == x for
// every x, zeros of both signs included), so the sums need no guards.  The
// sums share their first additions: message q's left-to-right sum starts
// with the payload plus the messages before q, which is also the start of
// every later message's sum, and continues one addition at a time with the
// messages after q.  Every message is therefore the canonical left-to-right
// sum itself, with nothing reassociated (no suffix sums, no subtraction),
// at DMAX^2/2 additions per coordinate instead of DMAX per message.
template <int R, int DMAX>
__global__ void __launch_bounds__(256) relaysum_pass_a_hub(RoundArgs a) {
    using T = RuleOf<R>;
    const bool ok[1] = {true};
    for (int h = blockIdx.y; h < a.nhubs; h += gridDim.y) {
        const int i = ldc(a.hubs + h);
        const int s0 = ldc(a.row_ptr + i);
        const int deg = ldc(a.row_ptr + i + 1) - s0;
        for (int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; c < a.nchunks;
             c += (int64_t)gridDim.x * blockDim.x) {
            const int64_t row = (int64_t)i * a.d + a.coff + a.cstride * c;
            lanev<1, 1> xv = zero_lane<1, 1>(), s1 = zero_lane<1, 1>(), s2 = zero_lane<1, 1>();
            if constexpr (T::reads_x) xv = load_lane<1, 1>(a.x + row, 0, ok);
            const lanev<1, 1> gv = load_lane<1, 1>(a.g + row, 0, ok);
            if constexpr (T::nesterov || T::adam) s1 = load_lane<1, 1>(a.s1 + row, 0, ok);
            if constexpr (T::adam) s2 = load_lane<1, 1>(a.s2 + row, 0, ok);
            float o[DMAX];
#pragma unroll
            for (int b = 0; b < DMAX; ++b)
                o[b] = b < deg ? load_float<true>(a.ring_prev + ring_off(a, hub_pos(a, ldc(a.rev + s0 + b)), c))
                               : -0.0f;
            const lanev<1, 1> p = payload<R, 1, 1>(a, xv, gv, s1, s2);
            if constexpr (T::nesterov || T::adam) store_lane<1, 1>(a.s1 + row, 0, ok, s1);
            if constexpr (T::adam) store_lane<1, 1>(a.s2 + row, 0, ok, s2);
            float pre = p.v[0][0];
#pragma unroll
            for (int q = 0; q < DMAX; ++q) {
                float m = pre;
#pragma unroll
                for (int b = q + 1; b < DMAX; ++b) m = m + o[b];
                if (q < deg) {
                    if (lost(a, s0 + q)) m = 0.0f;
                    store_float<true>(a.ring_next + ring_off(a, hub_pos(a, s0 + q), c), m);
                }
                pre = pre + o[q];
            }
            store_hub_payload<T>(a, i, row, c, p);
        }
    }
}

// Pass A for the workers of more than kHubDeg neighbours (a.hubs, a.nhubs),
// hub h in blockIdx.y, one carried coordinate per thread: the out-messages
// in blocks of kHubDeg, whose left-to-right sums stay in registers while the
// previous messages stream past once per block, each added to every sum of
// the block but its own message's (the canonical order, as in pass A).  A
// previous message is read ceil(deg / kHubDeg) times instead of deg - 1.
template <int R>
__global__ void __launch_bounds__(256) relaysum_pass_a_hub_big(RoundArgs a) {
    using T = RuleOf<R>;
    const bool ok[1] = {true};
    for (int h = blockIdx.y; h < a.nhubs; h += gridDim.y) {
        const int i = ldc(a.hubs + h);
        const int s0 = ldc(a.row_ptr + i);
        const int deg = ldc(a.row_ptr + i + 1) - s0;
        for (int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; c < a.nchunks;
             c += (int64_t)gridDim.x * blockDim.x) {
            const int64_t row = (int64_t)i * a.d + a.coff + a.cstride * c;
            lanev<1, 1> xv = zero_lane<1, 1>(), s1 = zero_lane<1, 1>(), s2 = zero_lane<1, 1>();
            if constexpr (T::reads_x) xv = load_lane<1, 1>(a.x + row, 0, ok);
            const lanev<1, 1> gv = load_lane<1, 1>(a.g + row, 0, ok);
            if constexpr (T::nesterov || T::adam) s1 = load_lane<1, 1>(a.s1 + row, 0, ok);
            if constexpr (T::adam) s2 = load_lane<1, 1>(a.s2 + row, 0, ok);
            const lanev<1, 1> p = payload<R, 1, 1>(a, xv, gv, s1, s2);
            if constexpr (T::nesterov || T::adam) store_lane<1, 1>(a.s1 + row, 0, ok, s1);
            if constexpr (T::adam) store_lane<1, 1>(a.s2 + row, 0, ok, s2);
            for (int q0 = 0; q0 < deg; q0 += kHubDeg) {
                float acc[kHubDeg];
#pragma unroll
                for (int j = 0; j < kHubDeg; ++j) acc[j] = p.v[0][0];
                for (int b = 0; b < deg; ++b) {
                    const float ob =
                        load_float<true>(a.ring_prev + ring_off(a, hub_pos(a, ldc(a.rev + s0 + b)), c));
                    if (b < q0 || b >= q0 + kHubDeg) {
#pragma unroll
                        for (int j = 0; j < kHubDeg; ++j) acc[j] = acc[j] + ob;
                    } else {
#pragma unroll
                        for (int j = 0; j < kHubDeg; ++j)
                            if (q0 + j != b) acc[j] = acc[j] + ob;
                    }
                }
#pragma unroll
                for (int j = 0; j < kHubDeg; ++j) {
                    const int q = q0 + j;
                    if (q < deg) {
                        const float m = lost(a, s0 + q) ? 0.0f : acc[j];
                        store_float<true>(a.ring_next + ring_off(a, hub_pos(a, s0 + q), c), m);
                    }
                }
            }
            store_hub_payload<T>(a, i, row, c, p);
        }
    }
}

// Pass B, worker blockIdx.y: new state from the payload and the new messages.
template <int C, int R>
__global__ void __launch_bounds__(256) relaysum_pass_b(RoundArgs a) {
    using T = RuleOf<R>;
    const bool ok[1] = {true};
    for (int i = blockIdx.y; i < a.n; i += gridDim.y) {
        const int s0 = a.row_ptr[i];
        const int deg = a.row_ptr[i + 1] - s0;
        const int nbar = a.nbar_out[i];
        const int64_t smp = T::mean ? a.smp_next[i] : (int64_t)1;
        for (int64_t chunk = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; chunk < a.nchunks;
             chunk += (int64_t)gridDim.x * blockDim.x) {
            const int64_t off = chunk * C;
            const int64_t row = (int64_t)i * a.d + a.coff + a.cstride * off;
            lanev<1, C> p, xo = zero_lane<1, C>();
            if constexpr (T::model) {
                p = load_lane<1, C>(a.x + row, 0, ok);          // the half-step from pass A
            } else if constexpr (T::robust) {
                xo = load_lane<1, C>(a.x + row, 0, ok);
                const lanev<1, C> gv = load_lane<1, C>(a.g + row, 0, ok);
                lanev<1, C> s1 = zero_lane<1, C>(), s2 = zero_lane<1, C>();
                if constexpr (T::nesterov || T::adam) s1 = load_lane<1, C>(a.s1 + row, 0, ok);
                if constexpr (T::adam) s2 = load_lane<1, C>(a.s2 + row, 0, ok);
                p = half_step_again<R, C>(a, xo, gv, s1, s2);
            } else if constexpr (T::grad) {
                xo = load_lane<1, C>(a.x + row, 0, ok);
                const lanev<1, C> gv = load_lane<1, C>(a.g + row, 0, ok);
                lanev<1, C> z1 = zero_lane<1, C>(), z2 = zero_lane<1, C>();
                p = payload<R, 1, C>(a, xo, gv, z1, z2);
            } else {
                p = load_lane<1, C>(a.g + row, 0, ok);
                xo = load_lane<1, C>(a.s1 + row, 0, ok);        // y
            }
            lanev<1, C> acc = p;
            for (int q = 0; q < deg; ++q)
                acc = add_lane<1, C>(acc, load_lane<1, C>(a.ring_next + ring_off(a, a.rev[s0 + q], off), 0, ok));
            const lanev<1, C> xn = new_state<R, 1, C>(a, acc, xo, nbar, smp);
            if constexpr (T::mean) store_lane<1, C>(a.s1 + row, 0, ok, xo);
            store_lane<1, C>(a.x + row, 0, ok, xn);
        }
    }
}

// ---- consensus distance ------------------------------------------------------

constexpr int kMetricBlocks = 1024;   // most blocks of the first stage

// Stage 1: block b takes coordinates b*256 + t, then a grid's width further
// on; per coordinate the mean of the n workers' values and the squared and
// absolute deviations from it, in binary64, summed (and maxed) per thread
// and then per block in a fixed tree order.  part[2b] = sum, part[2b+1] = max.
__global__ void __launch_bounds__(256) relaysum_consensus_kernel(const float *x, int32_t n,
                                                                 int64_t d, double *part) {
    __shared__ double s_sum[256];
    __shared__ double s_max[256];
    const int t = threadIdx.x;
    double acc = 0.0, mx = 0.0;
    for (int64_t c = (int64_t)blockIdx.x * 256 + t; c < d; c += (int64_t)gridDim.x * 256) {
        double mean = 0.0;
        for (int i = 0; i < n; ++i) mean += (double)x[(int64_t)i * d + c];
        mean /= (double)n;
        for (int i = 0; i < n; ++i) {
            const double e = (double)x[(int64_t)i * d + c] - mean;
            acc += e * e;
            mx = fmax(mx, fabs(e));
        }
    }
    s_sum[t] = acc;
    s_max[t] = mx;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if (t < w) {
            s_sum[t] += s_sum[t + w];
            s_max[t] = fmax(s_max[t], s_max[t + w]);
        }
        __syncthreads();
    }
    if (t == 0) {
        part[2 * blockIdx.x] = s_sum[0];
        part[2 * blockIdx.x + 1] = s_max[0];
    }
}

// Stage 2, one thread: the blocks' sums in block order, divided by n, and
// their maximum.
__global__ void __launch_bounds__(64) relaysum_consensus_final(const double *part, int nb, int32_t n,
                                                               double *out) {
    if (threadIdx.x != 0) return;
    double sum = 0.0, mx = 0.0;
    for (int b = 0; b < nb; ++b) {
        sum += part[2 * b];
        mx = fmax(mx, part[2 * b + 1]);
    }
    out[0] = sum / (double)n;
    out[1] = mx;
}

// ---- launch tables -----------------------------------------------------------

typedef void (*kernel_fn)(RoundArgs);
typedef void (*kernel2_fn)(RoundArgs, RoundArgs);

// Tile kernel: each lane streams U = 2 chunks of 4 floats per row and tile
// (a 2 KB tile row per wave), at most two workers per wave.  Rows need only
// 4-byte alignment and any d: 16-byte chunks at 4-byte alignment, the row's
// last d % 4 floats one by one.
constexpr int kU4 = 2;

template <int R, bool NT, bool TAIL, bool SP>
kernel_fn tile_for(int pw) {
    return pw == 1 ? relaysum_tile_kernel<kU4, 4, 1, R, NT, TAIL, SP>
                   : relaysum_tile_kernel<kU4, 4, 2, R, NT, TAIL, SP>;
}

template <int R, bool SP>
kernel_fn tile_for(int pw, bool nt, bool tail) {
    if (tail) return nt ? tile_for<R, true, true, SP>(pw) : tile_for<R, false, true, SP>(pw);
    return nt ? tile_for<R, true, false, SP>(pw) : tile_for<R, false, false, SP>(pw);
}

template <int R>
kernel_fn tile_for(int pw, bool nt, bool tail, bool sp) {
    return sp ? tile_for<R, true>(pw, nt, tail) : tile_for<R, false>(pw, nt, tail);
}

// Tile kernel of a rule; `tail` when d % 4 != 0 (the last chunk of every row
// is partial), `sp` with a spill sub-tile per workgroup.
kernel_fn pick_tile(int rule, int pw, bool nt, bool tail, bool sp = false) {
    if (pw != 1 && pw != 2) return nullptr;
    switch (rule) {
        case kModelSgd: return tile_for<kModelSgd>(pw, nt, tail, sp);
        case kModelNesterov: return tile_for<kModelNesterov>(pw, nt, tail, sp);
        case kModelAdam: return tile_for<kModelAdam>(pw, nt, tail, sp);
        case kRobustSgd: return tile_for<kRobustSgd>(pw, nt, tail, sp);
        case kRobustNesterov: return tile_for<kRobustNesterov>(pw, nt, tail, sp);
        case kRobustAdam: return tile_for<kRobustAdam>(pw, nt, tail, sp);
        case kGrad: return tile_for<kGrad>(pw, nt, tail, sp);
        case kMean: return tile_for<kMean>(pw, nt, tail, sp);
        default: return nullptr;
    }
}

template <int R>
void pass_for(kernel_fn *pa, kernel_fn *pb, kernel_fn *ph) {
    *pa = relaysum_pass_a<1, R>;
    *pb = relaysum_pass_b<1, R>;
    ph[0] = relaysum_pass_a_hub<R, 16>;
    ph[1] = relaysum_pass_a_hub<R, 32>;
    ph[2] = relaysum_pass_a_hub<R, 64>;
    ph[3] = relaysum_pass_a_hub_big<R>;
}

// Pass A, pass B (one carried coordinate per thread: the two-pass path
// takes double trees, whose coordinates of a tree are every second one) and
// the hub kernels of the degree classes of kHubClass, then the blocked one
// for the workers of more neighbours.
bool pick_passes(int rule, kernel_fn *pa, kernel_fn *pb, kernel_fn *ph) {
    switch (rule) {
        case kModelSgd: pass_for<kModelSgd>(pa, pb, ph); return true;
        case kModelNesterov: pass_for<kModelNesterov>(pa, pb, ph); return true;
        case kModelAdam: pass_for<kModelAdam>(pa, pb, ph); return true;
        case kRobustSgd: pass_for<kRobustSgd>(pa, pb, ph); return true;
        case kRobustNesterov: pass_for<kRobustNesterov>(pa, pb, ph); return true;
        case kRobustAdam: pass_for<kRobustAdam>(pa, pb, ph); return true;
        case kGrad: pass_for<kGrad>(pa, pb, ph); return true;
        case kMean: pass_for<kMean>(pa, pb, ph); return true;
        default: return false;
    }
}


template <int R>
kernel2_fn dtree_for(int pw, bool tail) {
    if (tail) return pw == 1 ? relaysum_dtree_kernel<1, R, true> : relaysum_dtree_kernel<2, R, true>;
    return pw == 1 ? relaysum_dtree_kernel<1, R, false> : relaysum_dtree_kernel<2, R, false>;
}

kernel2_fn pick_dtree(int rule, int pw, bool tail) {
    if (pw != 1 && pw != 2) return nullptr;
    switch (rule) {
        case kModelSgd: return dtree_for<kModelSgd>(pw, tail);
        case kModelNesterov: return dtree_for<kModelNesterov>(pw, tail);
        case kModelAdam: return dtree_for<kModelAdam>(pw, tail);
        case kRobustSgd: return dtree_for<kRobustSgd>(pw, tail);
        case kRobustNesterov: return dtree_for<kRobustNesterov>(pw, tail);
        case kRobustAdam: return dtree_for<kRobustAdam>(pw, tail);
        case kGrad: return dtree_for<kGrad>(pw, tail);
        case kMean: return dtree_for<kMean>(pw, tail);
        default: return nullptr;
    }
}

template <int R>
kernel2_fn dtree_seq_for(bool tail) {
    return tail ? relaysum_dtree_seq_kernel<4, R, true> : relaysum_dtree_seq_kernel<4, R, false>;
}

kernel2_fn pick_dtree_seq(int rule, int pw, bool tail) {
    if (pw > 4) return nullptr;
    switch (rule) {
        case kModelSgd: return dtree_seq_for<kModelSgd>(tail);
        case kModelNesterov: return dtree_seq_for<kModelNesterov>(tail);
        case kModelAdam: return dtree_seq_for<kModelAdam>(tail);
        case kRobustSgd: return dtree_seq_for<kRobustSgd>(tail);
        case kRobustNesterov: return dtree_seq_for<kRobustNesterov>(tail);
        case kRobustAdam: return dtree_seq_for<kRobustAdam>(tail);
        case kGrad: return dtree_seq_for<kGrad>(tail);
        case kMean: return dtree_seq_for<kMean>(tail);
        default: return nullptr;
    }
}

typedef void (*kernelc_fn)(RoundArgs, ClusterArgs);
typedef void (*kerneld_fn)(RoundArgs, RoundArgs, ClusterArgs, ClusterArgs);

template <int R>
void cluster_dtree_pair(bool tail, kerneld_fn *k1, kerneld_fn *k2) {
    *k1 = tail ? relaysum_cluster_dtree_kernel<2, R, true> : relaysum_cluster_dtree_kernel<2, R, false>;
    *k2 = tail ? relaysum_cluster_dtree_fixup<R, true> : relaysum_cluster_dtree_fixup<R, false>;
}

// Double-tree cluster kernels of a rule; the clusters hold 16 * pw workers,
// and pw = 2 is the one instantiated.
bool pick_cluster_dtree(int rule, bool tail, int pw, kerneld_fn *k1, kerneld_fn *k2) {
    if (pw != 2) return false;
    switch (rule) {
        case kModelSgd: cluster_dtree_pair<kModelSgd>(tail, k1, k2); return true;
        case kModelNesterov: cluster_dtree_pair<kModelNesterov>(tail, k1, k2); return true;
        case kModelAdam: cluster_dtree_pair<kModelAdam>(tail, k1, k2); return true;
        case kRobustSgd: cluster_dtree_pair<kRobustSgd>(tail, k1, k2); return true;
        case kRobustNesterov: cluster_dtree_pair<kRobustNesterov>(tail, k1, k2); return true;
        case kRobustAdam: cluster_dtree_pair<kRobustAdam>(tail, k1, k2); return true;
        case kGrad: cluster_dtree_pair<kGrad>(tail, k1, k2); return true;
        case kMean: cluster_dtree_pair<kMean>(tail, k1, k2); return true;
        default: return false;
    }
}

template <int R, bool NT, bool TAIL>
kernelc_fn cluster_for(bool low_degree, int pw) {
    if (low_degree) return relaysum_cluster_kernel<kU4, 4, kMaxDegInRegs, true, R, NT, TAIL, 1>;
    return pw == 2 ? relaysum_cluster_kernel<kU4, 4, kClusterDegInRegs, false, R, NT, TAIL, 2>
                   : relaysum_cluster_kernel<kU4, 4, kClusterDegInRegs, false, R, NT, TAIL, 1>;
}

template <int R>
void cluster_pair(bool low, int pw, bool nt, bool tail, bool c4, kernelc_fn *k1, kernelc_fn *k2) {
    if (tail) *k1 = nt ? cluster_for<R, true, true>(low, pw) : cluster_for<R, false, true>(low, pw);
    else *k1 = nt ? cluster_for<R, true, false>(low, pw) : cluster_for<R, false, false>(low, pw);
    *k2 = c4 ? relaysum_cluster_fixup<4, R> : relaysum_cluster_fixup<1, R>;
}

// Cluster kernel and boundary fixup of a rule; `tail` when d % 4 != 0, `c4`
// when the fixup may move whole 16-byte chunks (d % 4 == 0).
bool pick_cluster(int rule, bool low, int pw, bool nt, bool tail, bool c4, kernelc_fn *k1,
                  kernelc_fn *k2) {
    switch (rule) {
        case kModelSgd: cluster_pair<kModelSgd>(low, pw, nt, tail, c4, k1, k2); return true;
        case kModelNesterov: cluster_pair<kModelNesterov>(low, pw, nt, tail, c4, k1, k2); return true;
        case kModelAdam: cluster_pair<kModelAdam>(low, pw, nt, tail, c4, k1, k2); return true;
        case kRobustSgd: cluster_pair<kRobustSgd>(low, pw, nt, tail, c4, k1, k2); return true;
        case kRobustNesterov: cluster_pair<kRobustNesterov>(low, pw, nt, tail, c4, k1, k2); return true;
        case kRobustAdam: cluster_pair<kRobustAdam>(low, pw, nt, tail, c4, k1, k2); return true;
        case kGrad: cluster_pair<kGrad>(low, pw, nt, tail, c4, k1, k2); return true;
        case kMean: cluster_pair<kMean>(low, pw, nt, tail, c4, k1, k2); return true;
        default: return false;
    }
}

// LDS of the cluster kernel: sample counts (mean estimation), counters and
// nbar of the tree when it relays them, then the message tile of the
// largest cluster.
size_t cluster_lds_bytes(int n, int e2, int slots, bool mean, bool relay) {
    const size_t hdr =
        relay ? ((mean ? (size_t)n * 8 : 0) + ((size_t)e2 + n) * 4 + 15) & ~(size_t)15 : 0;
    return hdr + (size_t)slots * kWave * 4 * kU4 * sizeof(float);
}

// LDS of the double-tree kernel: both trees' counters, then two message tiles.
size_t dtree_lds_bytes(int n, int e2a, int e2b) {
    const size_t hdr = ((size_t)n * 16 + ((size_t)e2a + e2b + 2 * (size_t)n) * 4 + 15) & ~(size_t)15;
    return hdr + ((size_t)e2a + e2b) * kWave * kDTreeU * 2 * sizeof(float);
}

// LDS of the double-tree kernel that relays the trees one after the other:
// both trees' counters, then one message tile for the larger tree.
size_t dtree_seq_lds_bytes(int n, int e2a, int e2b) {
    const size_t hdr = ((size_t)n * 16 + ((size_t)e2a + e2b + 2 * (size_t)n) * 4 + 15) & ~(size_t)15;
    return hdr + (size_t)std::max(e2a, e2b) * kWave * kDTreeU * 2 * sizeof(float);
}


// LDS of the tile kernel: sample counts (mean estimation), counters and nbar,
// then the [2E][64 * floats_per_lane] message tile.
size_t tile_lds_bytes(int n, int e2, int floats_per_lane, bool mean) {
    const size_t hdr = ((mean ? (size_t)n * 8 : 0) + ((size_t)e2 + n) * 4 + 15) & ~(size_t)15;
    return hdr + (size_t)e2 * kWave * floats_per_lane * sizeof(float);
}

}  // namespace

// One tree of a handle: its CSR and counters.  A single-tree handle carries
// every coordinate on tree 0; a double-tree handle carries the odd
// coordinates on tree 0 (tree A) and the even ones on tree 1 (B).
struct TreeState : Csr {
    int32_t *d_topo = nullptr;    // row_ptr[n+1] | col[e2] | rev[e2] | src[e2] | hubs[nhubs]
    int32_t nhubs = 0;            // workers of more than kMaxDegInRegs2 neighbours,
    int32_t hub_class[kNumHubClasses] = {0, 0, 0, 0};   // listed by degree class (kHubClass, then
                                                         // more than kHubDeg), so many of each
    int32_t *d_counts = nullptr;  // cnt[2][e2] | nbar[n] | S[n]
    int64_t *d_samples = nullptr; // s_i for mean estimation, [2][n]
    int64_t len = 0;              // coordinates this tree carries
    int coff = 0;                 // first model coordinate it carries
    int cstride = 1;              // model-coordinate step between carried ones
    int32_t slot_base = 0;        // its first message slot in a ring tile
};

struct relaysum_s {
    int32_t n = 0;
    int64_t d = 0;
    int ntrees = 1;
    TreeState tr[2];
    // Message ring of all trees: [2][ring_tiles][ring_slots][2^ring_shift]
    // floats, parity t&1 written by round t.
    float *ring = nullptr;
    int64_t ring_tiles = 0;
    int32_t ring_slots = 0;
    int ring_shift = kRingShift;
    bool packed = false;          // lane-packed ring tiles (double trees)
    int64_t t = 0;
    // Mean estimation (Alg. 3): an upper bound, per tree, of every worker's
    // sample count s_i so far, and each tree's largest degree, from which
    // the bound grows (see nbar_bound).
    int64_t smp_bound[2] = {0, 0};
    int32_t max_deg[2] = {0, 0};
    hipStream_t stream = nullptr;
    int device = 0;
    // Device ranges that passed on_device(), most recent first: a round on
    // the arrays of the previous rounds checks nothing again.
    struct CheckedRange { const void *p = nullptr; size_t bytes = 0; } checked[8];
    int cu_count = 256;
    int waves = 1;               // W: waves per workgroup of the tile kernels
    int pw = 1;                  // workers per wave (power of two)
    bool tile = false;           // tile kernels (up to 32 workers) or two-pass path
    bool dseq = false;           // double trees of 33..64 workers: trees relayed in turn through LDS
    bool cluster = false;        // cluster kernels (single trees of more than 32 workers)
    int32_t cl_count = 0;        // clusters K
    int32_t cl_cap = 0;          // workers per cluster at most (one per wave)
    bool cl_relay = false;       // degrees <= kClusterLowDeg: counters relayed per workgroup
    bool cl_hubs = false;        // hub kernels ahead of the cluster kernel (workers of more
                                 //   than kMaxDegInRegs2 neighbours, in no cluster)
    bool dcluster = false;       // double trees of more than 64 workers as clusters
    int32_t cl_slots[2] = {0, 0};   // messages inside the largest cluster, per tree
    int32_t cl_nb = 0;           // boundary workers
    // members[K][cap] | lslot[2E] | bidx[n] | bnd[nb] | rpos[2E] | bfirst[nb]; on
    // double trees members | lslot A | lslot B | bidx | bnd | rpos A | rpos B |
    // bfirst A | bfirst B
    int32_t *d_cluster = nullptr;
    std::vector<int32_t> cl_rpos[2];   // ring position of each slot of each tree (cluster handles)
    float *cl_scratch = nullptr;    // partial sums of the boundary workers, [nb][d]
    double *d_metric = nullptr;     // consensus distance: block partials, then the result
    size_t lds_limit = 64 * 1024;   // LDS one workgroup may use
    size_t lds_cu = 160 * 1024;     // LDS of one CU (gfx950)
    struct Launch {
        kernel_fn fn = nullptr;
        kernel2_fn fn2 = nullptr;
        kernelc_fn fc1 = nullptr, fc2 = nullptr;
        kerneld_fn fd1 = nullptr, fd2 = nullptr;
        size_t lds = 0;
        int32_t spill = 0;       // tile kernel with a spill sub-tile: its coordinates
        int64_t spill_grid = 0;  //   per workgroup, and the workgroups
    } launch[2][kNumRules];      // [128-bit][rule], filled on first use
    std::string err;
};

static size_t ring_parity_floats(const relaysum_t *h) {
    return (size_t)h->ring_tiles * (size_t)h->ring_slots << h->ring_shift;
}

static int fail(relaysum_t *h, int code, const std::string &msg) {
    if (h) h->err = msg;
    return code;
}

static int hip_fail(relaysum_t *h, hipError_t e, const char *what) {
    return fail(h, RELAYSUM_ERR_DEVICE, std::string(what) + ": " + hipGetErrorString(e));
}

// The stream-ordered state calls (reset, poison, snapshots, accessors that
// synchronise) cannot be recorded into a graph: memset nodes and host
// synchronisation have no place in one.  Refuse them before anything is
// queued while the handle's stream is capturing.
static int refuse_capture(relaysum_t *h, const char *what) {
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    const hipError_t st = hipStreamIsCapturing(h->stream, &cs);
    if (st != hipSuccess) return hip_fail(h, st, what);
    if (cs != hipStreamCaptureStatusNone)
        return fail(h, RELAYSUM_ERR_INVALID_ARG,
                    std::string(what) + ": the handle's stream is capturing a graph");
    return RELAYSUM_OK;
}

static void release(relaysum_t *h) {
    if (!h) return;
    if (h->ring) (void)hipFree(h->ring);
    if (h->d_cluster) (void)hipFree(h->d_cluster);
    if (h->cl_scratch) (void)hipFree(h->cl_scratch);
    if (h->d_metric) (void)hipFree(h->d_metric);
    for (TreeState &tr : h->tr) {
        if (tr.d_samples) (void)hipFree(tr.d_samples);
        if (tr.d_counts) (void)hipFree(tr.d_counts);
        if (tr.d_topo) (void)hipFree(tr.d_topo);
    }
    delete h;
}

static int allocate_tree(relaysum_t *h, TreeState &tr) {
    const int n = h->n;
    std::vector<int32_t> hubs;
    for (int k = 0; k < kNumHubClasses; ++k) {
        const size_t before = hubs.size();
        const int lo = k == 0 ? kMaxDegInRegs2 : kHubClass[k - 1];
        const int hi = k < 3 ? kHubClass[k] : INT32_MAX;
        for (int32_t i = 0; i < n; ++i) {
            const int32_t deg = tr.row_ptr[i + 1] - tr.row_ptr[i];
            if (deg > lo && deg <= hi) hubs.push_back(i);
        }
        tr.hub_class[k] = (int32_t)(hubs.size() - before);
    }
    tr.nhubs = (int32_t)hubs.size();
    const size_t topo_ints = (size_t)(n + 1) + 3 * (size_t)tr.e2 + hubs.size();
    if (hipMalloc(&tr.d_topo, topo_ints * sizeof(int32_t)) != hipSuccess ||
        hipMalloc(&tr.d_counts, (2 * (size_t)tr.e2 + 2 * (size_t)n) * sizeof(int32_t)) != hipSuccess ||
        hipMalloc(&tr.d_samples, 2 * (size_t)n * sizeof(int64_t)) != hipSuccess) {
        (void)hipGetLastError();
        return RELAYSUM_ERR_OUT_OF_MEMORY;
    }
    std::vector<int32_t> topo;
    topo.reserve(topo_ints);
    topo.insert(topo.end(), tr.row_ptr.begin(), tr.row_ptr.end());
    topo.insert(topo.end(), tr.col.begin(), tr.col.end());
    topo.insert(topo.end(), tr.rev.begin(), tr.rev.end());
    topo.insert(topo.end(), tr.src.begin(), tr.src.end());
    topo.insert(topo.end(), hubs.begin(), hubs.end());
    if (hipMemcpy(tr.d_topo, topo.data(), topo_ints * sizeof(int32_t), hipMemcpyHostToDevice) !=
        hipSuccess)
        return RELAYSUM_ERR_DEVICE;
    return RELAYSUM_OK;
}

static int resolve_launch(relaysum_t *h, int rule, bool c4);

// Largest nbar_i any worker can have in round t of a tree of n workers whose
// degrees are at most deg: the workers within t + 1 hops (the counters of
// Alg. 1 count exactly those when no message is lost, fewer otherwise), at
// most 1 + deg * (1 + (deg-1) + ... + (deg-1)^t), and at most n.
static int64_t nbar_bound(int32_t n, int32_t deg, int64_t t) {
    if (deg <= 2) return std::min<int64_t>(n, 1 + (int64_t)deg * (t + 1));
    int64_t ball = 1, frontier = deg;
    for (int64_t hop = 0; hop <= t && ball < n; ++hop) {
        ball += frontier;
        frontier = std::min<int64_t>(frontier * (deg - 1), n);
    }
    return std::min<int64_t>(ball, n);
}

static int create_handle(int32_t n, int64_t d, const int32_t *const edges[2],
                         const int32_t num_edges[2], int ntrees, relaysum_t **out) {
    if (!out) return RELAYSUM_ERR_INVALID_ARG;
    *out = nullptr;
    if (n < 1 || n > RELAYSUM_MAX_WORKERS || d < 0) return RELAYSUM_ERR_INVALID_ARG;
    relaysum_t *h = new (std::nothrow) relaysum_s();
    if (!h) return RELAYSUM_ERR_OUT_OF_MEMORY;
    h->n = n;
    h->d = d;
    h->ntrees = ntrees;
    for (int k = 0; k < ntrees; ++k) {
        int rc;
        try {
            rc = build_csr(n, edges[k], num_edges[k], h->tr[k]);
        } catch (const std::bad_alloc &) {
            rc = RELAYSUM_ERR_OUT_OF_MEMORY;   // host memory for the CSR form
        }
        if (rc != RELAYSUM_OK) { release(h); return rc; }
    }
    for (int k = 0; k < ntrees; ++k)
        for (int32_t i = 0; i < n; ++i)
            h->max_deg[k] = std::max(h->max_deg[k], h->tr[k].row_ptr[i + 1] - h->tr[k].row_ptr[i]);
    if (ntrees == 1) {
        h->tr[0].len = d;
    } else {
        h->tr[0].len = d / 2;             // odd coordinates 1, 3, ...
        h->tr[0].coff = 1;
        h->tr[1].len = (d + 1) / 2;       // even coordinates 0, 2, ...
        h->tr[1].coff = 0;
        for (TreeState &tr : h->tr) tr.cstride = 2;
        h->tr[1].slot_base = h->tr[0].e2;
        h->packed = true;
    }
    int64_t longest = 0;
    for (int k = 0; k < ntrees; ++k) {
        h->ring_slots += h->tr[k].e2;
        longest = std::max(longest, h->tr[k].len);
    }

    hipError_t st = hipGetDevice(&h->device);
    if (st != hipSuccess) { release(h); return RELAYSUM_ERR_DEVICE; }
    int cus = 0, lds_max = 0, lds_cu = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, h->device) == hipSuccess &&
        cus > 0)
        h->cu_count = cus;
    if (hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, h->device) ==
            hipSuccess && lds_max > 0)
        h->lds_limit = (size_t)lds_max;
    if (hipDeviceGetAttribute(&lds_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor,
                              h->device) == hipSuccess && lds_cu > 0)
        h->lds_cu = (size_t)lds_cu;

    // Tile plan: W waves per workgroup, pw workers per wave.  Trees of up to
    // 32 workers use the tile kernels; larger ones the kernels below.  The
    // tile kernel stops at 32 workers because beyond that its [2E][64]-float
    // message tile fills LDS, leaving one workgroup per CU and 256-byte row
    // segments: on the 256-worker random tree it ran at 4.24 ms per round,
    // against 2.38 ms for the two-pass path.
    h->waves = std::min<int>(n, kMaxWaves);
    int pw = 1;
    while (pw * h->waves < n) pw *= 2;
    h->pw = pw;
    if (ntrees == 1)
        h->tile = pw <= 2 && tile_lds_bytes(n, h->tr[0].e2, 4 * kU4, true) <= h->lds_limit;
    else
        h->tile = pw <= 2 && dtree_lds_bytes(n, h->tr[0].e2, h->tr[1].e2) <= h->lds_limit;
    // Double trees of 33 to 64 workers relay one tree after the other
    // through one LDS message tile (126 KB at 64 workers).
    h->dseq = ntrees == 2 && !h->tile && pw <= 4 &&
              dtree_seq_lds_bytes(n, h->tr[0].e2, h->tr[1].e2) <= h->lds_limit;

    // Single trees of more than 32 workers run as clusters of at most 16
    // workers, provided the clusters are on average at least half full
    // (first-fit packing leaves at most one cluster half empty, so they are)
    // and the grid of (tile, cluster) workgroups fits one launch; other
    // trees take the two-pass path.
    // Trees of at most 256 workers and degree at most kClusterLowDeg (chains,
    // binary trees) relay the counters in every workgroup and run one
    // workgroup per CU on long grids, as the tile kernel does; the others
    // (random trees, larger trees, whose relay would walk thousands of
    // counters in every workgroup) take the counters from a launch before
    // and keep up to 8 previous messages per worker in registers.  On MI355X,
    // against the whole-tree-per-tile kernel these trees once took (since
    // removed: the two-pass path with hub kernels beat it 3 to 40 times on
    // every tree with a larger hub measured): chains of 33 to 256
    // workers 4-17% and binary trees of 63 to 256 workers 0-9% faster per
    // round; random trees of 100, 200 and 256 workers 1%, 5% and 6% faster.
    int32_t max_deg = 0, above_regs = 0;
    for (int32_t i = 0; i < n; ++i) {
        const int32_t deg = h->tr[0].row_ptr[i + 1] - h->tr[0].row_ptr[i];
        max_deg = std::max(max_deg, deg);
        above_regs += deg > kMaxDegInRegs2;   // the hub kernels' workers (allocate_tree lists them)
    }
    // Trees with a worker of more than kMaxDegInRegs2 neighbours plan their
    // clusters without those workers (the hubs): the hub kernels form the
    // hubs' payloads and out-messages in launches ahead of the cluster
    // kernel, one carried coordinate per thread with reads linear in the
    // degree, the members read the hubs' messages from the ring, and the
    // completion launch finishes the hubs' sums with the other boundary
    // workers'.  On MI355X, against the two-pass path these trees took
    // before, same box, bit for bit the same results: the pa2000
    // preferential-attachment tree (48 hubs) 2.96 -> 2.38 ms per round,
    // brooms of 200 workers with a hub of 41 1.79 -> 1.45 ms and of 2,000
    // with a hub of 501 5.25 -> 4.90 ms, stars of 256 workers the same; the
    // 1,000-worker broom with a hub of 13, whose hub re-read its
    // in-messages inside its cluster before, 2.16 -> 2.13 ms.
    ClusterPlan plan;
    const bool with_hubs = above_regs > 0;
    if (ntrees == 1 && !h->tile && d > 0) {
        const bool relay = max_deg <= kClusterLowDeg && n <= kMaxWaves * 16;
        const int cap = !relay && n >= kClusterPairFrom ? 2 * kMaxWaves : kMaxWaves;
        try {
            plan_clusters(n, h->tr[0], cap, plan, with_hubs ? kMaxDegInRegs2 : INT32_MAX);
        } catch (const std::bad_alloc &) {
            release(h);
            return RELAYSUM_ERR_OUT_OF_MEMORY;
        }
        if (plan.count > 0 && plan.nhubs == (with_hubs ? above_regs : 0) &&
            (int64_t)plan.count * cap <= 2 * (int64_t)(n - plan.nhubs) + cap &&
            (d + 511) / 512 * (int64_t)plan.count <= 0x7fffffff) {
            h->cluster = true;
            h->cl_hubs = plan.nhubs > 0;
            h->cl_count = plan.count;
            h->cl_cap = cap;
            h->cl_relay = relay;
            h->cl_slots[0] = plan.slots;
            h->cl_nb = (int32_t)plan.bnd.size();
            h->cl_rpos[0] = plan.rpos;
        }
    }
    // Double trees of more than 64 workers whose trees both have degrees of
    // at most kClusterMaxDeg run as clusters shared by both trees, under the
    // same conditions.
    DualPlan dplan;
    if (ntrees == 2 && !h->tile && !h->dseq && d > 0) {
        int32_t deg2 = 0;
        for (int k = 0; k < 2; ++k)
            for (int32_t i = 0; i < n; ++i)
                deg2 = std::max(deg2, h->tr[k].row_ptr[i + 1] - h->tr[k].row_ptr[i]);
        if (deg2 <= kClusterMaxDeg) {
            // Clusters of 32 workers, two per wave: half the boundary rows of
            // clusters of 16, and on MI355X 1-3% faster per round (the
            // 200-worker double binary trees at d = 1M 1.433 -> 1.39 ms, 128
            // workers at d = 3M 2.63 -> 2.60 ms); at 33 to 64 workers both
            // sizes were slower than the sequential double-tree kernel.
            const int cap = 2 * kMaxWaves;
            try {
                plan_clusters_dual(n, h->tr[0], h->tr[1], cap, dplan);
            } catch (const std::bad_alloc &) {
                release(h);
                return RELAYSUM_ERR_OUT_OF_MEMORY;
            }
            if ((int64_t)dplan.count * cap <= 2 * (int64_t)n + cap &&
                (d + 511) / 512 * (int64_t)dplan.count <= 0x7fffffff) {
                h->dcluster = true;
                h->cl_count = dplan.count;
                h->cl_cap = cap;
                h->cl_slots[0] = dplan.slots[0];
                h->cl_slots[1] = dplan.slots[1];
                h->cl_nb = (int32_t)dplan.bnd.size();
                h->cl_rpos[0] = dplan.rpos[0];
                h->cl_rpos[1] = dplan.rpos[1];
            }
        }
    }

    // Ring tiles hold 2^kRingShift floats of a message.  A shorter message
    // takes the smallest power of two that holds it, so that a slot costs
    // about its d floats rather than a whole ring tile: at 2^24 workers with
    // d = 5 the ring is 2 GB instead of 1 TB.  No kernel tile may straddle a
    // ring tile: 512 model coordinates in the tile, cluster and double-tree
    // kernels (and the 256-coordinate blocks of the packed double-tree
    // layout), one float on the two-pass path.  A message of at most 512
    // floats lies in one ring tile whatever its size, so single trees go
    // down to 4 floats; double trees keep 512 for the packed layout.
    // Single trees of more than 4096 directed edges (more than 2048 workers)
    // keep at most 512 floats per ring tile: a 4096-float ring tile of such
    // a tree spans more than 64 MB, with a workgroup's message pieces far
    // apart in it.  On MI355X the random tree of 8,192 workers at d = 40,000
    // took 2.44 instead of 2.60 ms per round that way, while trees of 256
    // and 1,000 workers measured the same and a chain of 64 workers 8-9%
    // slower with 512- or 1024-float ring tiles.
    const int shift_lo = ntrees == 1 ? 2 : 9;
    const int shift_hi = ntrees == 1 && h->ring_slots > 4096 ? 9 : kRingShift;
    int shift_fit = 0;
    while (shift_fit < shift_hi && ((int64_t)1 << shift_fit) < longest) ++shift_fit;
    h->ring_shift = std::max(shift_lo, shift_fit);
    h->ring_tiles = (longest + (((int64_t)1 << h->ring_shift) - 1)) >> h->ring_shift;

    for (int k = 0; k < ntrees; ++k) {
        int rc;
        try {
            rc = allocate_tree(h, h->tr[k]);
        } catch (const std::bad_alloc &) {
            rc = RELAYSUM_ERR_OUT_OF_MEMORY;   // host staging of the topology
        }
        if (rc != RELAYSUM_OK) { release(h); return rc; }
    }
    if (h->ring_slots > 0 && h->ring_tiles > 0 &&
        hipMalloc(&h->ring, 2 * ring_parity_floats(h) * sizeof(float)) != hipSuccess) {
        (void)hipGetLastError();
        release(h);
        return RELAYSUM_ERR_OUT_OF_MEMORY;
    }
    if (h->cluster || h->dcluster) {
        std::vector<int32_t> tab;
        if (h->cluster) {
            tab.reserve(plan.members.size() + plan.lslot.size() + plan.bidx.size() + plan.bnd.size() +
                        plan.rpos.size() + plan.bfirst.size());
            for (const std::vector<int32_t> *v : {&plan.members, &plan.lslot, &plan.bidx, &plan.bnd,
                                                  &plan.rpos, &plan.bfirst})
                tab.insert(tab.end(), v->begin(), v->end());
        } else {
            for (const std::vector<int32_t> *v :
                 {&dplan.members, &dplan.lslot[0], &dplan.lslot[1], &dplan.bidx, &dplan.bnd,
                  &dplan.rpos[0], &dplan.rpos[1], &dplan.bfirst[0], &dplan.bfirst[1]})
                tab.insert(tab.end(), v->begin(), v->end());
        }
        if (hipMalloc(&h->d_cluster, tab.size() * sizeof(int32_t)) != hipSuccess ||
            (h->cl_nb > 0 &&
             hipMalloc(&h->cl_scratch, (size_t)h->cl_nb * (size_t)d * sizeof(float)) != hipSuccess)) {
            (void)hipGetLastError();
            release(h);
            return RELAYSUM_ERR_OUT_OF_MEMORY;
        }
        if (hipMemcpy(h->d_cluster, tab.data(), tab.size() * sizeof(int32_t),
                      hipMemcpyHostToDevice) != hipSuccess) {
            release(h);
            return RELAYSUM_ERR_DEVICE;
        }
    }
    if (relaysum_reset(h) != RELAYSUM_OK || hipStreamSynchronize(h->stream) != hipSuccess) {
        release(h);
        return RELAYSUM_ERR_DEVICE;
    }
    for (int c4 = 0; c4 < 2; ++c4)
        for (int rule = 0; rule < kNumRules; ++rule) {
            const int rc = resolve_launch(h, rule, c4 != 0);
            if (rc != RELAYSUM_OK) {
                release(h);
                return rc;
            }
        }
    *out = h;
    return RELAYSUM_OK;
}

// Tree and slot within it of a handle-wide (tree-major) slot number.
static bool locate_slot(const relaysum_t *h, int32_t slot, int *tree, int32_t *local) {
    if (slot < 0) return false;
    for (int k = 0; k < h->ntrees; ++k) {
        if (slot < h->tr[k].e2) {
            *tree = k;
            *local = slot;
            return true;
        }
        slot -= h->tr[k].e2;
    }
    return false;
}

// Kernel path of a round of this handle.  Every path takes any 4-byte
// aligned rows.
enum Path { kPathTile, kPathDTree, kPathCluster, kPathTwoPass, kPathDTreeSeq, kPathClusterDTree };

static Path path_of(const relaysum_t *h) {
    if (h->tile && h->ntrees == 1) return kPathTile;
    if (h->tile) return kPathDTree;
    if (h->dseq && h->d > 0) return kPathDTreeSeq;
    if (h->dcluster && h->d > 0) return kPathClusterDTree;
    if (h->cluster && h->d > 0 && h->ntrees == 1) return kPathCluster;
    return kPathTwoPass;
}

// Kernel and dynamic LDS of `rule` on this handle (single-kernel paths).
// relaysum_create resolves every rule, so that a round only launches kernels
// and can be captured into a HIP graph.  The kernel's dynamic-LDS limit is
// set to the device maximum rather than to this handle's need: the
// attribute belongs to the kernel, which other handles share.
static int resolve_launch(relaysum_t *h, int rule, bool c4) {
    relaysum_s::Launch &L = h->launch[c4][rule];
    const bool mean = rule == kMean;
    const bool adam = rule == kModelAdam || rule == kRobustAdam;
    const bool uses_s1 = adam || mean || rule == kModelNesterov || rule == kRobustNesterov;
    // Residency cap of 16 waves per CU on long grids: the launch reserves
    // enough LDS that at most 16/W workgroups fit on a CU.  On the 16-worker
    // chain two co-resident 16-wave workgroups streamed 3-6% slower than one
    // (more concurrent DRAM streams per CU for the same bytes in flight).  A
    // short grid (under 8 tiles per CU) is bound by its last dispatch round
    // instead, and runs without the cap: the 16-worker heap at d = 270,000
    // (528 tiles) took 30.6 instead of 32.9 us per round.
    const int per_cu = std::max(1, kMaxWaves / h->waves);
    const int64_t grid_tiles =
        (h->d + 511) / 512 *
        (path_of(h) == kPathCluster || path_of(h) == kPathClusterDTree ? h->cl_count : 1);   // workgroups
    const size_t cap_lds = grid_tiles >= 8 * (int64_t)h->cu_count
                               ? std::min(h->lds_cu / (size_t)(per_cu + 1) + 256, h->lds_limit)
                               : 0;
    const void *fn = nullptr;
    size_t lds = 0;
    switch (path_of(h)) {
        case kPathTile: {
            // Cache-allocating accesses when the round's working set (the
            // rows it reads or writes and both ring parities) takes at most
            // half of the 256 MB MALL, so that the next round finds it there:
            // on the 16-worker heap at d = 270,000 (117 MB) a round took
            // 27.5-29.0 us instead of 30.6-31.4 us.  Larger rounds stream past
            // the caches (on the 16-worker chain at d = 9.75M cache-allocating
            // accesses took 1.09 ms per round instead of 0.93 ms).
            const size_t rows = 2 + (uses_s1 ? 1 : 0) + (adam ? 1 : 0);
            const size_t working_set =
                (rows * (size_t)h->n * (size_t)h->d + 2 * ring_parity_floats(h)) * sizeof(float);
            const bool nt = working_set > kMallBytes / 2;
            L.fn = pick_tile(rule, h->pw, nt, h->d % 4 != 0);
            fn = (const void *)L.fn;
            const int floats_per_lane = 4 * kU4;
            lds = std::max(tile_lds_bytes(h->n, h->tr[0].e2, floats_per_lane, mean), cap_lds);
            // A short grid whose tiles exceed a whole number of dispatch rounds
            // (G workgroups, k rounds of the R resident at once) by at most
            // 64 coordinates per resident workgroup spreads the excess over
            // the first round's workgroups (spill sub-tiles of a power of two
            // of at most 64 coordinates, so none straddles a ring tile; the
            // later workgroups' spills are empty) instead of running one more
            // round.  Each round with spills pays for their latency chain
            // once: spread over all G workgroups, a 16-worker tree at
            // d = 398,216 (three rounds of 256) took 64.5 instead of 52.6 us.
            const bool keeps_old = rule == kRobustSgd || rule == kRobustNesterov ||
                                   rule == kRobustAdam || rule == kGrad || mean;
            const size_t lds_sp =
                tile_lds_bytes(h->n, h->tr[0].e2, floats_per_lane, mean) +
                ((size_t)h->tr[0].e2 + (size_t)h->n * (keeps_old ? 2 : 1)) * kWave * sizeof(float);
            const kernel_fn fn_sp = pick_tile(rule, h->pw, nt, h->d % 4 != 0, true);
            int per_cu_sp = 0;
            if (cap_lds == 0 && h->d > 512 * (int64_t)h->cu_count && lds_sp <= h->lds_limit) {
                hipError_t st = hipFuncSetAttribute((const void *)fn_sp,
                                                    hipFuncAttributeMaxDynamicSharedMemorySize,
                                                    (int)h->lds_limit);
                if (st == hipSuccess)
                    st = hipOccupancyMaxActiveBlocksPerMultiprocessor(
                        &per_cu_sp, (const void *)fn_sp, h->waves * kWave, lds_sp);
                if (st != hipSuccess) return hip_fail(h, st, "tile kernel occupancy");
            }
            const int64_t resident = (int64_t)per_cu_sp * h->cu_count;
            const int64_t G = resident > 0 ? h->d / 512 / resident * resident : 0;
            const int64_t left = h->d - G * 512;
            const int64_t ring_tile = (int64_t)1 << h->ring_shift;
            if (G > 0 && G % 16 == 0 && left > 0 && left <= resident * kWave &&
                (G * 512) % ring_tile == 0) {
                int64_t sp = 1;
                while (sp * resident < left) sp *= 2;
                if (ring_tile % sp == 0) {
                    L.fn = fn_sp;
                    fn = (const void *)L.fn;
                    L.spill = (int32_t)sp;
                    L.spill_grid = G;
                    lds = lds_sp;
                }
            }
            break;
        }
        case kPathDTree:
            L.fn2 = pick_dtree(rule, h->pw, h->d % 4 != 0);
            fn = (const void *)L.fn2;
            lds = std::max(dtree_lds_bytes(h->n, h->tr[0].e2, h->tr[1].e2), cap_lds);
            break;
        case kPathDTreeSeq:
            L.fn2 = pick_dtree_seq(rule, h->pw, h->d % 4 != 0);
            fn = (const void *)L.fn2;
            lds = std::max(dtree_seq_lds_bytes(h->n, h->tr[0].e2, h->tr[1].e2), cap_lds);
            break;
        case kPathCluster: {
            const size_t rows = 2 + (uses_s1 ? 1 : 0) + (adam ? 1 : 0);
            const size_t working_set =
                (rows * (size_t)h->n * (size_t)h->d + 2 * ring_parity_floats(h)) * sizeof(float);
            if (!pick_cluster(rule, h->cl_relay, h->cl_cap / kMaxWaves, working_set > kMallBytes / 2,
                              h->d % 4 != 0,
                              h->d % 4 == 0, &L.fc1, &L.fc2))
                return fail(h, RELAYSUM_ERR_INVALID_ARG, "no cluster kernel for this rule");
            fn = (const void *)L.fc1;
            lds = cluster_lds_bytes(h->n, h->tr[0].e2, h->cl_slots[0], mean, h->cl_relay);
            if (h->cl_relay) lds = std::max(lds, cap_lds);
            break;
        }
        case kPathClusterDTree:
            if (!pick_cluster_dtree(rule, h->d % 4 != 0, h->cl_cap / kMaxWaves, &L.fd1, &L.fd2))
                return fail(h, RELAYSUM_ERR_INVALID_ARG, "no cluster kernel for this rule");
            fn = (const void *)L.fd1;
            // Both trees' message tiles of the largest cluster; no residency cap.
            lds = ((size_t)h->cl_slots[0] + h->cl_slots[1]) * kWave * kDTreeU * 2 * sizeof(float);
            break;
        case kPathTwoPass:
            return RELAYSUM_OK;   // fixed launches without dynamic LDS
    }
    if (!fn) return fail(h, RELAYSUM_ERR_INVALID_ARG, "no kernel for this tree and rule");
    if (lds > h->lds_limit) return fail(h, RELAYSUM_ERR_INVALID_ARG, "tree too large for LDS");
    hipError_t st = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize,
                                        (int)h->lds_limit);
    if (st != hipSuccess) return hip_fail(h, st, "hipFuncSetAttribute");
    L.lds = lds;
    return RELAYSUM_OK;
}

extern "C" {

const char *relaysum_strerror(int code) {
    switch (code) {
        case RELAYSUM_OK: return "ok";
        case RELAYSUM_ERR_INVALID_ARG: return "invalid argument";
        case RELAYSUM_ERR_NOT_A_TREE: return "edge list is not a tree on n workers";
        case RELAYSUM_ERR_OUT_OF_MEMORY: return "out of memory";
        case RELAYSUM_ERR_DEVICE: return "HIP device error";
        default: return "unknown status";
    }
}

const char *relaysum_last_error(const relaysum_t *h) { return h ? h->err.c_str() : g_static_err; }

int relaysum_create(int32_t n, int64_t d, const int32_t *edges, int32_t num_edges,
                    relaysum_t **out) {
    const int32_t *e[2] = {edges, nullptr};
    const int32_t ne[2] = {num_edges, 0};
    return create_handle(n, d, e, ne, 1, out);
}

int relaysum_create_double(int32_t n, int64_t d, const int32_t *edges_a, const int32_t *edges_b,
                           int32_t num_edges, relaysum_t **out) {
    const int32_t *e[2] = {edges_a, edges_b};
    const int32_t ne[2] = {num_edges, num_edges};
    return create_handle(n, d, e, ne, 2, out);
}

int relaysum_destroy(relaysum_t *h) {
    if (!h) return RELAYSUM_OK;
    const hipError_t st = hipStreamSynchronize(h->stream);
    release(h);
    return st == hipSuccess ? RELAYSUM_OK : RELAYSUM_ERR_DEVICE;
}

int relaysum_set_stream(relaysum_t *h, void *hip_stream) {
    if (!h) return RELAYSUM_ERR_INVALID_ARG;
    h->stream = reinterpret_cast<hipStream_t>(hip_stream);
    return RELAYSUM_OK;
}

int relaysum_reset(relaysum_t *h) {
    if (!h) return RELAYSUM_ERR_INVALID_ARG;
    if (const int rc = refuse_capture(h, "reset")) return rc;
    hipError_t st = hipSuccess;
    for (int k = 0; k < h->ntrees && st == hipSuccess; ++k) {
        TreeState &tr = h->tr[k];
        st = hipMemsetAsync(tr.d_counts, 0, (2 * (size_t)tr.e2 + 2 * (size_t)h->n) * sizeof(int32_t), h->stream);
        if (st == hipSuccess)
            st = hipMemsetAsync(tr.d_samples, 0, 2 * (size_t)h->n * sizeof(int64_t), h->stream);
    }
    if (st == hipSuccess && h->ring)
        st = hipMemsetAsync(h->ring, 0, 2 * ring_parity_floats(h) * sizeof(float), h->stream);
    if (st != hipSuccess) return hip_fail(h, st, "reset");
    h->t = 0;
    h->smp_bound[0] = h->smp_bound[1] = 0;
    return RELAYSUM_OK;
}

int relaysum_round(const relaysum_t *h, int64_t *t) {
    if (!h || !t) return RELAYSUM_ERR_INVALID_ARG;
    *t = h->t;
    return RELAYSUM_OK;
}

int relaysum_kernel_path(const relaysum_t *h, int32_t *path) {
    if (!h || !path) return RELAYSUM_ERR_INVALID_ARG;
    switch (path_of(h)) {
        case kPathTile: *path = RELAYSUM_PATH_TILE; break;
        case kPathDTree: *path = RELAYSUM_PATH_DTREE; break;
        case kPathCluster: *path = RELAYSUM_PATH_CLUSTER; break;
        case kPathTwoPass: *path = RELAYSUM_PATH_TWO_PASS; break;
        case kPathDTreeSeq: *path = RELAYSUM_PATH_DTREE_SEQ; break;
        case kPathClusterDTree: *path = RELAYSUM_PATH_CLUSTER_DTREE; break;
    }
    return RELAYSUM_OK;
}

int relaysum_num_trees(const relaysum_t *h, int32_t *count) {
    if (!h || !count) return RELAYSUM_ERR_INVALID_ARG;
    *count = h->ntrees;
    return RELAYSUM_OK;
}

int relaysum_num_directed_edges(const relaysum_t *h, int32_t *count) {
    if (!h || !count) return RELAYSUM_ERR_INVALID_ARG;
    int32_t c = 0;
    for (int k = 0; k < h->ntrees; ++k) c += h->tr[k].e2;
    *count = c;
    return RELAYSUM_OK;
}

int relaysum_directed_edge(const relaysum_t *h, int32_t slot, int32_t *src, int32_t *dst) {
    int k;
    int32_t s;
    if (!h || !locate_slot(h, slot, &k, &s)) return RELAYSUM_ERR_INVALID_ARG;
    if (src) *src = h->tr[k].src[s];
    if (dst) *dst = h->tr[k].col[s];
    return RELAYSUM_OK;
}

int relaysum_message_length(const relaysum_t *h, int32_t slot, int64_t *len) {
    int k;
    int32_t s;
    if (!h || !len || !locate_slot(h, slot, &k, &s)) return RELAYSUM_ERR_INVALID_ARG;
    *len = h->tr[k].len;
    return RELAYSUM_OK;
}

// Whether the bytes [p, p + bytes) lie in device memory (or managed memory)
// of GPU `device`, within one allocation: host memory, another GPU's memory
// or a buffer shorter than the round's rows would make a kernel fault.
// hipPointerGetAttributes gives the memory's kind and GPU,
// hipMemGetAddressRange the allocation that holds p (memory it cannot place,
// such as mappings made with the virtual-memory calls, passes on its kind
// and GPU alone); neither allocates.
static bool on_device(const void *p, size_t bytes, int device) {
    hipPointerAttribute_t at;
    if (hipPointerGetAttributes(&at, p) != hipSuccess) {
        (void)hipGetLastError();
        return false;
    }
    if (at.type != hipMemoryTypeDevice && at.type != hipMemoryTypeManaged) return false;
    if (at.type == hipMemoryTypeDevice && at.device != device) return false;
    hipDeviceptr_t base = nullptr;
    size_t size = 0;
    if (hipMemGetAddressRange(&base, &size, const_cast<void *>(p)) != hipSuccess || !base) {
        (void)hipGetLastError();
        return true;
    }
    const uintptr_t b = (uintptr_t)base, q = (uintptr_t)p;
    return q >= b && q - b <= size && bytes <= size - (q - b);
}

// on_device() through the handle's cache of ranges already checked.
static bool on_device_cached(relaysum_t *h, const void *p, size_t bytes) {
    for (const auto &c : h->checked)
        if (c.p == p && c.bytes >= bytes) return true;
    if (!on_device(p, bytes, h->device)) return false;
    for (int k = 7; k > 0; --k) h->checked[k] = h->checked[k - 1];
    h->checked[0].p = p;
    h->checked[0].bytes = bytes;
    return true;
}

// Kernel arguments of tree k for this round.
static RoundArgs tree_args(const relaysum_t *h, int k, const RoundArgs &common) {
    const TreeState &tr = h->tr[k];
    const int prev = (int)((h->t + 1) & 1), next = (int)(h->t & 1);
    RoundArgs a = common;
    const size_t slot0 = (size_t)tr.slot_base << h->ring_shift;
    a.ring_prev = h->ring ? h->ring + (size_t)prev * ring_parity_floats(h) + slot0 : nullptr;
    a.ring_next = h->ring ? h->ring + (size_t)next * ring_parity_floats(h) + slot0 : nullptr;
    a.cnt_prev = tr.d_counts + (size_t)prev * tr.e2;
    a.cnt_next = tr.d_counts + (size_t)next * tr.e2;
    a.nbar_out = tr.d_counts + 2 * (size_t)tr.e2;
    a.cnt_sum = a.nbar_out + h->n;
    a.smp_prev = tr.d_samples + (size_t)prev * h->n;
    a.smp_next = tr.d_samples + (size_t)next * h->n;
    a.row_ptr = tr.d_topo;
    a.col = tr.d_topo + h->n + 1;
    a.rev = a.col + tr.e2;
    a.src = a.rev + tr.e2;
    a.hubs = a.src + tr.e2;
    a.nhubs = tr.nhubs;
    a.e2 = tr.e2;
    a.ring_shift = h->ring_shift;
    a.ring_packed = h->packed ? 1 : 0;
    a.ring_slots = h->ring_slots;
    a.cstride = tr.cstride;
    a.coff = tr.coff;
    return a;
}

int relaysum_step_ex(relaysum_t *h, float *x, const float *g, float *state1, float *state2,
                     const relaysum_round_args *args) {
    if (!h) return RELAYSUM_ERR_INVALID_ARG;
    if (!args) return fail(h, RELAYSUM_ERR_INVALID_ARG, "args is NULL");
    const bool adam = args->optimizer == RELAYSUM_OPT_ADAM;
    if (args->optimizer != RELAYSUM_OPT_SGD && !adam)
        return fail(h, RELAYSUM_ERR_INVALID_ARG, "unknown optimizer");
    int rule = -1;
    switch (args->update) {
        case RELAYSUM_UPDATE_MODEL:
            rule = adam ? kModelAdam : (args->beta1 != 0.0f ? kModelNesterov : kModelSgd);
            break;
        case RELAYSUM_UPDATE_ROBUST:
            rule = adam ? kRobustAdam : (args->beta1 != 0.0f ? kRobustNesterov : kRobustSgd);
            break;
        case RELAYSUM_UPDATE_GRAD:
            if (adam || args->beta1 != 0.0f)
                return fail(h, RELAYSUM_ERR_INVALID_ARG, "the Grad rule takes plain SGD updates");
            rule = kGrad;
            break;
        case RELAYSUM_UPDATE_MEAN:
            if (adam || args->beta1 != 0.0f)
                return fail(h, RELAYSUM_ERR_INVALID_ARG, "mean estimation has no optimizer");
            rule = kMean;
            break;
        default:
            return fail(h, RELAYSUM_ERR_INVALID_ARG, "unknown update rule");
    }
    if (adam && args->adam_step < 1) return fail(h, RELAYSUM_ERR_INVALID_ARG, "adam_step < 1");
    const bool need_s1 = rule == kModelNesterov || rule == kRobustNesterov || adam || rule == kMean;
    const bool need_s2 = adam;
    if (h->d > 0) {
        if (!x || !g) return fail(h, RELAYSUM_ERR_INVALID_ARG, "x and g must not be NULL");
        if (need_s1 && !state1) return fail(h, RELAYSUM_ERR_INVALID_ARG, "state1 is NULL");
        if (need_s2 && !state2) return fail(h, RELAYSUM_ERR_INVALID_ARG, "state2 is NULL");
    }
    const uintptr_t bits = (uintptr_t)x | (uintptr_t)g | (need_s1 ? (uintptr_t)state1 : 0) |
                           (need_s2 ? (uintptr_t)state2 : 0);
    if (h->d > 0 && (bits & 3))
        return fail(h, RELAYSUM_ERR_INVALID_ARG, "x, g and state rows must be 4-byte aligned");
    if (h->d > 0) {
        // Workers' rows are read and rewritten tile by tile, so arrays that
        // share bytes would mix one round's inputs with its outputs.
        const size_t bytes = (size_t)h->n * (size_t)h->d * sizeof(float);
        const uintptr_t arr[4] = {(uintptr_t)x, (uintptr_t)g,
                                  need_s1 ? (uintptr_t)state1 : 0, need_s2 ? (uintptr_t)state2 : 0};
        for (int i = 0; i < 4; ++i)
            for (int j = i + 1; j < 4; ++j)
                if (arr[i] && arr[j] && arr[i] < arr[j] + bytes && arr[j] < arr[i] + bytes)
                    return fail(h, RELAYSUM_ERR_INVALID_ARG, "x, g and state arrays overlap");
        const char *name[4] = {"x", "g", "state1", "state2"};
        for (int i = 0; i < 4; ++i)
            if (arr[i] && !on_device_cached(h, (const void *)arr[i], bytes))
                return fail(h, RELAYSUM_ERR_INVALID_ARG,
                            std::string(name[i]) +
                                " is not n*d floats of device memory on the handle's GPU");
    }
    if (args->dropped) {
        size_t slots = 0;
        for (int k = 0; k < h->ntrees; ++k) slots += (size_t)h->tr[k].e2;
        if (slots > 0 && !on_device_cached(h, args->dropped, slots))
            return fail(h, RELAYSUM_ERR_INVALID_ARG,
                        "dropped is not one byte per directed edge of device memory on the handle's GPU");
    }

    RoundArgs c;
    std::memset(&c, 0, sizeof c);
    c.x = x;
    c.g = g;
    c.s1 = need_s1 ? state1 : nullptr;
    c.s2 = need_s2 ? state2 : nullptr;
    c.d = h->d;
    c.n = h->n;
    c.lr = args->lr;
    c.beta1 = args->beta1;
    c.beta2 = args->beta2;
    c.eps = args->eps;
    c.one_m_b1 = 1.0f - args->beta1;
    c.one_m_b2 = 1.0f - args->beta2;
    c.step_size = 0.0f;
    c.bc2_sqrt = 1.0f;
    if (adam) {
        // PyTorch's bias corrections, in double, each rounded once to binary32.
        const double bc1 = 1.0 - std::pow((double)args->beta1, (double)args->adam_step);
        const double bc2 = 1.0 - std::pow((double)args->beta2, (double)args->adam_step);
        c.step_size = (float)((double)args->lr / bc1);
        c.bc2_sqrt = (float)std::sqrt(bc2);
    }
    RoundArgs ta[2];
    for (int k = 0; k < h->ntrees; ++k) {
        ta[k] = tree_args(h, k, c);
        ta[k].dropped = args->dropped ? args->dropped + (k == 0 ? 0 : h->tr[0].e2) : nullptr;
    }

    const bool c4 = (h->d % 4 == 0) && (bits & 15) == 0;
    const bool mean = rule == kMean;
    // Alg. 3 divides y_i by the integer s_i converted to binary32, exact up
    // to 2^24: refuse a round that could take some s_i past it.
    int64_t smp_after[2] = {h->smp_bound[0], h->smp_bound[1]};
    if (mean) {
        for (int k = 0; k < h->ntrees; ++k) {
            smp_after[k] += nbar_bound(h->n, h->max_deg[k], h->t);
            if (smp_after[k] > ((int64_t)1 << 24))
                return fail(h, RELAYSUM_ERR_INVALID_ARG,
                            "mean estimation: this round could take a worker's sample count past "
                            "2^24, where its binary32 divisor is no longer exact");
        }
    }
    const int threads = h->waves * kWave;
    const Path path = path_of(h);
    const relaysum_s::Launch &L = h->launch[c4][rule];
    if (path != kPathTwoPass && !L.fn && !L.fn2 && !L.fc1 && !L.fd1) {
        const int rc = resolve_launch(h, rule, c4);
        if (rc != RELAYSUM_OK) return rc;
    }

    if (path == kPathTile) {
        RoundArgs &a = ta[0];
        a.nchunks = h->d / 4;                                   // whole 16-byte chunks
        a.ntiles = (h->d + kWave * kU4 * 4 - 1) / (kWave * kU4 * 4);
        // One workgroup per tile (d == 0: one workgroup still relays the
        // counters); with a spill, whole dispatch rounds only.
        const int64_t grid = L.spill ? L.spill_grid : std::max<int64_t>(a.ntiles, 1);
        a.spill = L.spill;
        a.spill_base = L.spill ? L.spill_grid * kWave * kU4 * 4 : 0;
        if (grid > 0x7fffffff) return fail(h, RELAYSUM_ERR_INVALID_ARG, "d too large");
        hipLaunchKernelGGL(L.fn, dim3((unsigned)grid), dim3(threads), L.lds, h->stream, a);
        hipError_t st = hipGetLastError();
        if (st != hipSuccess) return hip_fail(h, st, "tile kernel launch");
    } else if (path == kPathDTree || path == kPathDTreeSeq) {
        // Double trees, 128-bit rows: one kernel relays both trees.  Its tile
        // is 64 * kDTreeU float4 chunks of the model (256 carried coordinates
        // per tree).
        for (int k = 0; k < 2; ++k) {
            ta[k].nchunks = h->d / 4;   // whole chunks; a partial last one with d % 4 != 0
            ta[k].ntiles = (h->d + kWave * kDTreeU * 4 - 1) / (kWave * kDTreeU * 4);
        }
        const int64_t grid = std::max<int64_t>(ta[0].ntiles, 1);
        if (grid > 0x7fffffff) return fail(h, RELAYSUM_ERR_INVALID_ARG, "d too large");
        hipLaunchKernelGGL(L.fn2, dim3((unsigned)grid), dim3(threads), L.lds, h->stream, ta[0],
                           ta[1]);
        hipError_t st = hipGetLastError();
        if (st != hipSuccess) return hip_fail(h, st, "double-tree kernel launch");
    } else if (path == kPathCluster) {
        RoundArgs &a = ta[0];
        a.nchunks = h->d / 4;                                   // whole 16-byte chunks
        a.ntiles = (h->d + kWave * kU4 * 4 - 1) / (kWave * kU4 * 4);
        const int64_t grid = a.ntiles * h->cl_count;
        if (grid > 0x7fffffff) return fail(h, RELAYSUM_ERR_INVALID_ARG, "d too large");
        ClusterArgs k;
        k.members = h->d_cluster;
        k.lslot = k.members + (size_t)h->cl_count * h->cl_cap;
        k.bidx = k.lslot + h->tr[0].e2;
        k.bnd = k.bidx + h->n;
        k.rpos = k.bnd + h->cl_nb;
        k.bfirst = k.rpos + h->tr[0].e2;
        k.scratch = h->cl_scratch;
        k.count = h->cl_count;
        k.cap = h->cl_cap;
        k.slots = h->cl_slots[0];
        k.nb = h->cl_nb;
        if (!h->cl_relay) {
            const unsigned cg = (unsigned)((h->tr[0].e2 + (int64_t)h->n + 255) / 256);
            if (h->cl_hubs) {
                hipLaunchKernelGGL(relaysum_count_sums_kernel, dim3((unsigned)((h->n + 255) / 256)),
                                   dim3(256), 0, h->stream, a);
                hipLaunchKernelGGL(relaysum_count_grid_kernel<true>, dim3(cg), dim3(256), 0, h->stream, a,
                                   mean ? 1 : 0);
            } else {
                hipLaunchKernelGGL(relaysum_count_grid_kernel<false>, dim3(cg), dim3(256), 0, h->stream, a,
                                   mean ? 1 : 0);
            }
        }
        if (h->cl_hubs) {
            // The hubs' payloads (into their scratch rows) and out-messages
            // (at the plan's ring positions), one carried coordinate per
            // thread, a launch per degree class.
            kernel_fn pa = nullptr, pb = nullptr, ph[kNumHubClasses] = {nullptr, nullptr, nullptr, nullptr};
            if (!pick_passes(rule, &pa, &pb, ph)) return fail(h, RELAYSUM_ERR_INVALID_ARG, "rule");
            RoundArgs ah = a;
            ah.nchunks = h->d;
            ah.hub_rpos = k.rpos;
            ah.hub_pay = k.scratch;
            ah.hub_bidx = k.bidx;
            for (int c = 0; c < kNumHubClasses; ++c) {
                ah.nhubs = h->tr[0].hub_class[c];
                if (ah.nhubs > 0) {
                    const unsigned hx = (unsigned)std::min<int64_t>((ah.nchunks + 255) / 256, 1024);
                    const unsigned hy = (unsigned)std::min<int64_t>(ah.nhubs, 65535);
                    hipLaunchKernelGGL(ph[c], dim3(hx, hy), dim3(256), 0, h->stream, ah);
                }
                ah.hubs += ah.nhubs;
            }
        }
        hipLaunchKernelGGL(L.fc1, dim3((unsigned)grid), dim3(threads), L.lds, h->stream, a, k);
        hipError_t st = hipGetLastError();
        if (st != hipSuccess) return hip_fail(h, st, "cluster kernel launch");
        if (h->cl_nb > 0) {
            // Boundary workers: C floats per thread, C = 4 when rows hold
            // whole 16-byte chunks.
            RoundArgs b = a;
            b.nchunks = h->d % 4 == 0 ? h->d / 4 : h->d;
            const unsigned gx = (unsigned)std::min<int64_t>((b.nchunks + 255) / 256, 1024);
            const unsigned gy = (unsigned)std::min<int64_t>(h->cl_nb, 65535);
            hipLaunchKernelGGL(L.fc2, dim3(gx, gy), dim3(256), 0, h->stream, b, k);
            st = hipGetLastError();
            if (st != hipSuccess) return hip_fail(h, st, "cluster fixup launch");
        }
    } else if (path == kPathClusterDTree) {
        for (int k = 0; k < 2; ++k) {
            ta[k].nchunks = h->d / 4;   // whole chunks; a partial last one with d % 4 != 0
            ta[k].ntiles = (h->d + kWave * kDTreeU * 4 - 1) / (kWave * kDTreeU * 4);
        }
        const int64_t grid = ta[0].ntiles * h->cl_count;
        if (grid > 0x7fffffff) return fail(h, RELAYSUM_ERR_INVALID_ARG, "d too large");
        const size_t e2a = h->tr[0].e2, e2b = h->tr[1].e2;
        ClusterArgs ka, kb;
        ka.members = kb.members = h->d_cluster;
        ka.lslot = ka.members + (size_t)h->cl_count * h->cl_cap;
        kb.lslot = ka.lslot + e2a;
        ka.bidx = kb.bidx = kb.lslot + e2b;
        ka.bnd = kb.bnd = ka.bidx + h->n;
        ka.rpos = ka.bnd + h->cl_nb;
        kb.rpos = ka.rpos + e2a;
        ka.bfirst = kb.rpos + e2b;
        kb.bfirst = ka.bfirst + h->cl_nb;
        ka.scratch = kb.scratch = h->cl_scratch;
        ka.count = kb.count = h->cl_count;
        ka.cap = kb.cap = h->cl_cap;
        ka.slots = h->cl_slots[0];
        kb.slots = h->cl_slots[1];
        ka.nb = kb.nb = h->cl_nb;
        const unsigned cg = (unsigned)((e2a + e2b + 2 * (int64_t)h->n + 255) / 256);
        hipLaunchKernelGGL(relaysum_count_grid2_kernel, dim3(cg), dim3(256), 0, h->stream, ta[0], ta[1],
                           mean ? 1 : 0);
        hipLaunchKernelGGL(L.fd1, dim3((unsigned)grid), dim3(threads), L.lds, h->stream, ta[0], ta[1], ka, kb);
        hipError_t st = hipGetLastError();
        if (st != hipSuccess) return hip_fail(h, st, "double-tree cluster kernel launch");
        if (h->cl_nb > 0) {
            const unsigned gx = (unsigned)std::min<int64_t>((ta[0].ntiles * 64 + 255) / 256, 1024);
            const unsigned gy = (unsigned)std::min<int64_t>(h->cl_nb, 65535);
            hipLaunchKernelGGL(L.fd2, dim3(gx, gy), dim3(256), 0, h->stream, ta[0], ta[1], ka, kb);
            st = hipGetLastError();
            if (st != hipSuccess) return hip_fail(h, st, "double-tree cluster fixup launch");
        }
    } else {
        // Two-pass path, one tree at a time.  The trees of a double-tree
        // handle own disjoint coordinates (stride 2), so their passes do not
        // interact; their rows are read one float per lane.  (Single trees
        // get here with d == 0, the counters alone, or when the cluster
        // grid would not fit one launch.)
        kernel_fn pa = nullptr, pb = nullptr, ph[kNumHubClasses] = {nullptr, nullptr, nullptr, nullptr};
        if (!pick_passes(rule, &pa, &pb, ph)) return fail(h, RELAYSUM_ERR_INVALID_ARG, "rule");
        for (int k = 0; k < h->ntrees; ++k) {
            RoundArgs &a = ta[k];
            a.nchunks = h->tr[k].len;
            a.ntiles = 0;
            hipLaunchKernelGGL(relaysum_count_kernel, dim3(1), dim3(1024), 0, h->stream, a,
                               mean ? 1 : 0);
            if (a.nchunks > 0) {
                const int64_t want = (a.nchunks + 255) / 256;
                const unsigned gx = (unsigned)std::min<int64_t>(want, 1024);
                const unsigned gy = (unsigned)std::min<int64_t>(h->n, 65535);
                hipLaunchKernelGGL(pa, dim3(gx, gy), dim3(256), 0, h->stream, a);
                // The hub workers, one carried coordinate per thread, a launch
                // per degree class.
                RoundArgs ah = a;
                ah.nchunks = h->tr[k].len;
                for (int c = 0; c < kNumHubClasses; ++c) {
                    ah.nhubs = h->tr[k].hub_class[c];
                    if (ah.nhubs > 0) {
                        const unsigned hx = (unsigned)std::min<int64_t>((ah.nchunks + 255) / 256, 1024);
                        const unsigned hy = (unsigned)std::min<int64_t>(ah.nhubs, 65535);
                        hipLaunchKernelGGL(ph[c], dim3(hx, hy), dim3(256), 0, h->stream, ah);
                    }
                    ah.hubs += ah.nhubs;
                }
                hipLaunchKernelGGL(pb, dim3(gx, gy), dim3(256), 0, h->stream, a);
            }
            hipError_t st = hipGetLastError();
            if (st != hipSuccess) return hip_fail(h, st, "two-pass launch");
        }
    }
    h->t += 1;
    h->smp_bound[0] = smp_after[0];
    h->smp_bound[1] = smp_after[1];
    return RELAYSUM_OK;
}

int relaysum_step(relaysum_t *h, float *x, const float *g, float *mom, float lr, float beta) {
    if (!h) return RELAYSUM_ERR_INVALID_ARG;
    if (beta != 0.0f && !mom && h->d > 0)
        return fail(h, RELAYSUM_ERR_INVALID_ARG, "mom is NULL but beta != 0");
    relaysum_round_args args;
    std::memset(&args, 0, sizeof args);
    args.update = RELAYSUM_UPDATE_MODEL;
    args.optimizer = RELAYSUM_OPT_SGD;
    args.lr = lr;
    args.beta1 = beta;
    return relaysum_step_ex(h, x, g, mom, nullptr, &args);
}

int relaysum_get_counts(relaysum_t *h, int32_t *nbar_host, int32_t *edge_counts_host) {
    if (!h) return RELAYSUM_ERR_INVALID_ARG;
    if (const int rc = refuse_capture(h, "get_counts")) return rc;
    const int last = (int)((h->t + 1) & 1);   // slot written by round t-1
    hipError_t st = hipSuccess;
    for (int k = 0; k < h->ntrees && st == hipSuccess; ++k) {
        const TreeState &tr = h->tr[k];
        if (edge_counts_host && tr.e2 > 0)
            st = hipMemcpyAsync(edge_counts_host + (k ? h->tr[0].e2 : 0),
                                tr.d_counts + (size_t)last * tr.e2, tr.e2 * sizeof(int32_t),
                                hipMemcpyDeviceToHost, h->stream);
        if (st == hipSuccess && nbar_host)
            st = hipMemcpyAsync(nbar_host + (size_t)k * h->n, tr.d_counts + 2 * (size_t)tr.e2,
                                h->n * sizeof(int32_t), hipMemcpyDeviceToHost, h->stream);
    }
    if (st == hipSuccess) st = hipStreamSynchronize(h->stream);
    return st == hipSuccess ? RELAYSUM_OK : hip_fail(h, st, "get_counts");
}

int relaysum_get_samples(relaysum_t *h, int64_t *samples_host) {
    if (!h || !samples_host) return RELAYSUM_ERR_INVALID_ARG;
    if (const int rc = refuse_capture(h, "get_samples")) return rc;
    const int last = (int)((h->t + 1) & 1);
    hipError_t st = hipSuccess;
    for (int k = 0; k < h->ntrees && st == hipSuccess; ++k)
        st = hipMemcpyAsync(samples_host + (size_t)k * h->n,
                            h->tr[k].d_samples + (size_t)last * h->n, h->n * sizeof(int64_t),
                            hipMemcpyDeviceToHost, h->stream);
    if (st == hipSuccess) st = hipStreamSynchronize(h->stream);
    return st == hipSuccess ? RELAYSUM_OK : hip_fail(h, st, "get_samples");
}

int relaysum_consensus_distance(relaysum_t *h, const float *x, double *dist, double *spread) {
    if (!h || !dist) return RELAYSUM_ERR_INVALID_ARG;
    if (const int rc = refuse_capture(h, "consensus_distance")) return rc;
    if (h->d == 0) {
        *dist = 0.0;
        if (spread) *spread = 0.0;
        return RELAYSUM_OK;
    }
    if (!x || ((uintptr_t)x & 3))
        return fail(h, RELAYSUM_ERR_INVALID_ARG, "consensus_distance: x is NULL or not 4-byte aligned");
    if (!on_device_cached(h, x, (size_t)h->n * (size_t)h->d * sizeof(float)))
        return fail(h, RELAYSUM_ERR_INVALID_ARG,
                    "consensus_distance: x is not n*d floats of device memory on the handle's GPU");
    if (!h->d_metric &&
        hipMalloc(&h->d_metric, (2 * (size_t)kMetricBlocks + 2) * sizeof(double)) != hipSuccess) {
        (void)hipGetLastError();
        h->d_metric = nullptr;
        return fail(h, RELAYSUM_ERR_OUT_OF_MEMORY, "consensus_distance: device buffer");
    }
    const int nb = (int)std::min<int64_t>((h->d + 255) / 256, kMetricBlocks);
    double *out = h->d_metric + 2 * (size_t)kMetricBlocks;
    hipLaunchKernelGGL(relaysum_consensus_kernel, dim3(nb), dim3(256), 0, h->stream, x, h->n, h->d,
                       h->d_metric);
    hipLaunchKernelGGL(relaysum_consensus_final, dim3(1), dim3(64), 0, h->stream,
                       (const double *)h->d_metric, nb, h->n, out);
    double res[2] = {0.0, 0.0};
    hipError_t st = hipGetLastError();
    if (st == hipSuccess)
        st = hipMemcpyAsync(res, out, sizeof res, hipMemcpyDeviceToHost, h->stream);
    if (st == hipSuccess) st = hipStreamSynchronize(h->stream);
    if (st != hipSuccess) return hip_fail(h, st, "consensus_distance");
    *dist = res[0];
    if (spread) *spread = res[1];
    return RELAYSUM_OK;
}

// ---- snapshots ----------------------------------------------------------------

}  // extern "C"

namespace {

// Header of a state snapshot.  The blocks after it: per tree the last
// round's counters (one int32 per slot), nbar (int32 per worker) and sample
// counts (int64 per worker); then the ring parity the next round reads,
// [ring tiles][slots][2^ring_shift] floats with the slots in CSR order
// (tree-major).  The cluster kernels keep each cluster's messages side by
// side in the ring instead; their slots are permuted to and from CSR order
// on the way, so a snapshot does not depend on the kernel path that wrote
// it.  Version 1 stored the ring in the kernel path's order; version 2 had no
// bound of the sample counts.
struct StateHeader {
    char magic[8];
    uint32_t version;
    int32_t n;
    int64_t d;
    int32_t ntrees;
    int32_t ring_shift;
    int64_t ring_tiles;
    int32_t ring_slots;
    int32_t packed;
    int64_t t;
    uint64_t tree_digest;
    int32_t e2[2];
    int64_t smp_bound[2];   // the handle's bound of the sample counts (mean estimation)
};
constexpr char kStateMagic[8] = {'R', 'L', 'Y', 'S', 'U', 'M', 'S', 'T'};
constexpr uint32_t kStateVersion = 3;

// FNV-1a over the trees' CSR form: handles built from the same trees (in
// any edge order) agree.
uint64_t tree_digest(const relaysum_t *h) {
    uint64_t x = 1469598103934665603ull;
    auto mix = [&](int64_t v) {
        for (int b = 0; b < 8; ++b) {
            x ^= (uint64_t)((v >> (8 * b)) & 0xff);
            x *= 1099511628211ull;
        }
    };
    mix(h->n);
    mix(h->ntrees);
    for (int k = 0; k < h->ntrees; ++k) {
        for (int32_t v : h->tr[k].row_ptr) mix(v);
        for (int32_t v : h->tr[k].col) mix(v);
    }
    return x;
}

StateHeader state_header(const relaysum_t *h) {
    StateHeader hd;
    std::memset(&hd, 0, sizeof hd);
    std::memcpy(hd.magic, kStateMagic, sizeof hd.magic);
    hd.version = kStateVersion;
    hd.n = h->n;
    hd.d = h->d;
    hd.ntrees = h->ntrees;
    hd.ring_shift = h->ring_shift;
    hd.ring_tiles = h->ring ? h->ring_tiles : 0;
    hd.ring_slots = h->ring_slots;
    hd.packed = h->packed ? 1 : 0;
    hd.t = h->t;
    hd.smp_bound[0] = h->smp_bound[0];
    hd.smp_bound[1] = h->smp_bound[1];
    hd.tree_digest = tree_digest(h);
    for (int k = 0; k < h->ntrees; ++k) hd.e2[k] = h->tr[k].e2;
    return hd;
}

size_t state_bytes(const relaysum_t *h) {
    size_t b = sizeof(StateHeader);
    for (int k = 0; k < h->ntrees; ++k)
        b += (size_t)h->tr[k].e2 * 4 + (size_t)h->n * 4 + (size_t)h->n * 8;
    if (h->ring) b += ring_parity_floats(h) * sizeof(float);
    return b;
}

// Copies between the snapshot's blocks and the handle's device buffers, in
// snapshot order, queued on the handle's stream.
hipError_t state_blocks(relaysum_t *h, unsigned char *snap, bool save) {
    const int last = (int)((h->t + 1) & 1);
    size_t off = sizeof(StateHeader);
    hipError_t st = hipSuccess;
    auto move = [&](void *dev, size_t nbytes) {
        if (st != hipSuccess || nbytes == 0) return;
        st = save ? hipMemcpyAsync(snap + off, dev, nbytes, hipMemcpyDefault, h->stream)
                  : hipMemcpyAsync(dev, snap + off, nbytes, hipMemcpyDefault, h->stream);
        off += nbytes;
    };
    for (int k = 0; k < h->ntrees; ++k) {
        TreeState &tr = h->tr[k];
        move(tr.d_counts + (size_t)last * tr.e2, (size_t)tr.e2 * 4);
        move(tr.d_counts + 2 * (size_t)tr.e2, (size_t)h->n * 4);
        move(tr.d_samples + (size_t)last * h->n, (size_t)h->n * 8);
    }
    if (h->ring) {
        float *ring = h->ring + (size_t)last * ring_parity_floats(h);
        if (!h->cluster && !h->dcluster) {
            move(ring, ring_parity_floats(h) * sizeof(float));
        } else if (st == hipSuccess) {
            // Slot s of tree k at ring position slot_base + cl_rpos[k][s] <->
            // position slot_base + s of the snapshot: one strided copy of its
            // ring-tile pieces per slot.
            const size_t piece = ((size_t)1 << h->ring_shift) * sizeof(float);
            const size_t pitch = (size_t)h->ring_slots * piece;
            unsigned char *snap_ring = snap + off;
            for (int k = 0; k < h->ntrees; ++k) {
                const size_t sb = (size_t)h->tr[k].slot_base;
                for (int32_t s = 0; s < h->tr[k].e2 && st == hipSuccess; ++s) {
                    unsigned char *dev =
                        reinterpret_cast<unsigned char *>(ring) + (sb + (size_t)h->cl_rpos[k][s]) * piece;
                    unsigned char *cpy = snap_ring + (sb + (size_t)s) * piece;
                    st = save ? hipMemcpy2DAsync(cpy, pitch, dev, pitch, piece, (size_t)h->ring_tiles,
                                                 hipMemcpyDefault, h->stream)
                              : hipMemcpy2DAsync(dev, pitch, cpy, pitch, piece, (size_t)h->ring_tiles,
                                                 hipMemcpyDefault, h->stream);
                }
            }
            off += ring_parity_floats(h) * sizeof(float);
        }
    }
    if (st == hipSuccess) st = hipStreamSynchronize(h->stream);
    return st;
}

}  // namespace

extern "C" {

int relaysum_state_size(const relaysum_t *h, size_t *bytes) {
    if (!h || !bytes) return RELAYSUM_ERR_INVALID_ARG;
    *bytes = state_bytes(h);
    return RELAYSUM_OK;
}

int relaysum_save_state(relaysum_t *h, void *buf, size_t bytes) {
    if (!h) return RELAYSUM_ERR_INVALID_ARG;
    if (const int rc = refuse_capture(h, "save_state")) return rc;
    if (!buf) return fail(h, RELAYSUM_ERR_INVALID_ARG, "save_state: buf is NULL");
    if (bytes < state_bytes(h))
        return fail(h, RELAYSUM_ERR_INVALID_ARG, "save_state: buffer smaller than relaysum_state_size");
    const StateHeader hd = state_header(h);
    hipError_t st = hipMemcpyAsync(buf, &hd, sizeof hd, hipMemcpyDefault, h->stream);
    if (st == hipSuccess) st = state_blocks(h, static_cast<unsigned char *>(buf), true);
    return st == hipSuccess ? RELAYSUM_OK : hip_fail(h, st, "save_state");
}

int relaysum_load_state(relaysum_t *h, const void *buf, size_t bytes) {
    if (!h) return RELAYSUM_ERR_INVALID_ARG;
    if (const int rc = refuse_capture(h, "load_state")) return rc;
    if (!buf) return fail(h, RELAYSUM_ERR_INVALID_ARG, "load_state: buf is NULL");
    if (bytes < sizeof(StateHeader))
        return fail(h, RELAYSUM_ERR_INVALID_ARG, "load_state: buffer shorter than a snapshot header");
    StateHeader hd;
    hipError_t st = hipMemcpyAsync(&hd, buf, sizeof hd, hipMemcpyDefault, h->stream);
    if (st == hipSuccess) st = hipStreamSynchronize(h->stream);
    if (st != hipSuccess) return hip_fail(h, st, "load_state");
    StateHeader mine = state_header(h);
    mine.t = hd.t;
    mine.smp_bound[0] = hd.smp_bound[0];
    mine.smp_bound[1] = hd.smp_bound[1];
    if (std::memcmp(hd.magic, kStateMagic, sizeof hd.magic) != 0 || hd.version != kStateVersion)
        return fail(h, RELAYSUM_ERR_INVALID_ARG, "load_state: not a snapshot of this library version");
    if (std::memcmp(&hd, &mine, sizeof hd) != 0 || hd.t < 0)
        return fail(h, RELAYSUM_ERR_INVALID_ARG,
                    "load_state: snapshot of a handle with other workers, model length or trees");
    if (bytes < state_bytes(h))
        return fail(h, RELAYSUM_ERR_INVALID_ARG, "load_state: buffer shorter than the snapshot");
    if (hd.smp_bound[0] < 0 || hd.smp_bound[1] < 0 || hd.smp_bound[0] > ((int64_t)1 << 24) ||
        hd.smp_bound[1] > ((int64_t)1 << 24))
        return fail(h, RELAYSUM_ERR_INVALID_ARG, "load_state: sample-count bound out of range");
    const int64_t t_before = h->t;
    h->t = hd.t;   // selects the parity the blocks go to
    st = state_blocks(h, static_cast<unsigned char *>(const_cast<void *>(buf)), false);
    if (st != hipSuccess) {
        h->t = t_before;
        return hip_fail(h, st, "load_state");
    }
    h->smp_bound[0] = hd.smp_bound[0];
    h->smp_bound[1] = hd.smp_bound[1];
    return RELAYSUM_OK;
}

int relaysum_poison_next(relaysum_t *h) {
    if (!h) return RELAYSUM_ERR_INVALID_ARG;
    if (const int rc = refuse_capture(h, "poison_next")) return rc;
    const int next = (int)(h->t & 1);
    hipError_t st = hipSuccess;
    for (int k = 0; k < h->ntrees && st == hipSuccess; ++k) {
        TreeState &tr = h->tr[k];
        st = hipMemsetAsync(tr.d_counts + (size_t)next * tr.e2, 0xff, (size_t)tr.e2 * 4, h->stream);
        if (st == hipSuccess)   // nbar and the counter sums
            st = hipMemsetAsync(tr.d_counts + 2 * (size_t)tr.e2, 0xff, 2 * (size_t)h->n * 4, h->stream);
        if (st == hipSuccess)
            st = hipMemsetAsync(tr.d_samples + (size_t)next * h->n, 0xff, (size_t)h->n * 8, h->stream);
    }
    if (st == hipSuccess && h->ring)
        st = hipMemsetAsync(h->ring + (size_t)next * ring_parity_floats(h), 0xff,
                            ring_parity_floats(h) * sizeof(float), h->stream);
    if (st == hipSuccess && h->cl_scratch)   // the partial sums of the boundary workers
        st = hipMemsetAsync(h->cl_scratch, 0xff, (size_t)h->cl_nb * (size_t)h->d * sizeof(float),
                            h->stream);
    return st == hipSuccess ? RELAYSUM_OK : hip_fail(h, st, "poison_next");
}

int relaysum_get_message(relaysum_t *h, int32_t slot, float *dst_host) {
    int k;
    int32_t s;
    if (!h || !dst_host || !locate_slot(h, slot, &k, &s)) return RELAYSUM_ERR_INVALID_ARG;
    if (const int rc = refuse_capture(h, "get_message")) return rc;
    const TreeState &tr = h->tr[k];
    if (tr.len == 0) return RELAYSUM_OK;
    const int last = (int)((h->t + 1) & 1);
    // Gather the message's ring-tile pieces out of the tile-major ring.
    const int64_t rt = (int64_t)1 << h->ring_shift;
    const int32_t pos = tr.slot_base + (h->cluster || h->dcluster ? h->cl_rpos[k][s] : s);
    const float *first = h->ring + (size_t)last * ring_parity_floats(h) + ((size_t)pos << h->ring_shift);
    const size_t pitch = (size_t)h->ring_slots * rt * sizeof(float);
    hipError_t st = hipSuccess;
    if (h->packed) {
        // Whole ring tiles of the message, then the lane-packed order undone.
        const int64_t tiles = (tr.len + rt - 1) / rt;
        std::vector<float> raw;
        try {
            raw.resize((size_t)tiles * rt);
        } catch (const std::bad_alloc &) {
            return fail(h, RELAYSUM_ERR_OUT_OF_MEMORY, "get_message: host staging buffer");
        }
        st = hipMemcpy2DAsync(raw.data(), rt * sizeof(float), first, pitch, rt * sizeof(float),
                              (size_t)tiles, hipMemcpyDeviceToHost, h->stream);
        if (st == hipSuccess) st = hipStreamSynchronize(h->stream);
        if (st != hipSuccess) return hip_fail(h, st, "get_message");
        for (int64_t c = 0; c < tr.len; ++c)
            dst_host[c] = raw[(size_t)((c & ~(rt - 1)) + packed_pos(c & (rt - 1)))];
        return RELAYSUM_OK;
    }
    const int64_t full = tr.len / rt, rem = tr.len % rt;
    if (full > 0)
        st = hipMemcpy2DAsync(dst_host, rt * sizeof(float), first, pitch, rt * sizeof(float),
                              (size_t)full, hipMemcpyDeviceToHost, h->stream);
    if (st == hipSuccess && rem > 0)
        st = hipMemcpyAsync(dst_host + full * rt, first + (size_t)full * h->ring_slots * rt,
                            rem * sizeof(float), hipMemcpyDeviceToHost, h->stream);
    if (st == hipSuccess) st = hipStreamSynchronize(h->stream);
    return st == hipSuccess ? RELAYSUM_OK : hip_fail(h, st, "get_message");
}

}  // extern "C"

// ---- the entry point that allocates nothing ------------------------------------
//
// relaysum_step_static runs relaysum_step's round for trees of up to
// kStaticMaxWorkers workers (the tile kernel's range) without a handle: the
// state a handle would allocate (the tree's CSR form, the two counter
// parities, nbar and the two ring parities) lives in one file-scope device
// array.  Each GPU holds its own copy of the array for the life of the
// process; its device address comes from hipGetSymbolAddress, taken once per
// device on the first call there (the array's name in host code is only a
// host-side stand-in).  Round t == 0 writes the tree and clears the counter
// and ring parity that round 0 reads with one fill kernel (no memset node,
// so the call can be recorded into a graph); later rounds find round t-1's
// state in the array.  Calls on one GPU share the array: overlapping runs
// race, and a new run (t == 0) replaces the previous one.

namespace {

constexpr int kStaticMaxWorkers = 32;
constexpr size_t kStaticBytes = (size_t)64 << 20;   // 64 MiB per GPU
constexpr int kStaticMaxDevices = 64;

static __device__ __align__(256) unsigned char static_scratch[kStaticBytes];

struct StaticTopo {
    int32_t n, e2;
    int32_t row_ptr[kStaticMaxWorkers + 1];
    int32_t col[2 * (kStaticMaxWorkers - 1)];
    int32_t rev[2 * (kStaticMaxWorkers - 1)];
    int32_t src[2 * (kStaticMaxWorkers - 1)];
};

// Round 0 of a run: the tree's CSR form into the array, the counter parity
// round 0 reads cleared (workgroup 0), and the ring parity it reads cleared
// (every workgroup, grid-strided, 16 bytes per access: a ring parity holds
// whole ring tiles of at least 512 floats).
__global__ void __launch_bounds__(256) relaysum_static_prepare(StaticTopo tp, int32_t *topo,
                                                               int32_t *cnt_prev, f4_t *ring_prev,
                                                               int64_t ring_f4) {
    if (blockIdx.x == 0) {
        const int topo_ints = tp.n + 1 + 3 * tp.e2;
        for (int k = threadIdx.x; k < topo_ints; k += blockDim.x) {
            int32_t v;
            if (k <= tp.n) v = tp.row_ptr[k];
            else if (k <= tp.n + tp.e2) v = tp.col[k - tp.n - 1];
            else if (k <= tp.n + 2 * tp.e2) v = tp.rev[k - tp.n - 1 - tp.e2];
            else v = tp.src[k - tp.n - 1 - 2 * tp.e2];
            topo[k] = v;
        }
        for (int s = threadIdx.x; s < tp.e2; s += blockDim.x) cnt_prev[s] = 0;
    }
    const f4_t z = {0.0f, 0.0f, 0.0f, 0.0f};
    for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < ring_f4;
         k += (int64_t)gridDim.x * blockDim.x)
        ring_prev[k] = z;
}

// What the static entry point remembers per device: the array's address and
// the run whose state it holds.
struct StaticDevice {
    unsigned char *base = nullptr;   // device address of static_scratch on this GPU
    int cu_count = 256;
    size_t lds_limit = 64 * 1024, lds_cu = 160 * 1024;
    bool run = false;                // a run's state is in the array
    int32_t n = 0;
    int64_t d = 0;
    uint64_t digest = 0;
    int64_t next_t = 0;
    const void *checked[3] = {nullptr, nullptr, nullptr};   // x, g, mom of the last call that passed
    size_t checked_bytes = 0;
};

StaticDevice g_static[kStaticMaxDevices];
std::mutex g_static_mu;

int static_fail(int code, const char *msg) {
    std::snprintf(g_static_err, sizeof g_static_err, "relaysum_step_static: %s", msg);
    return code;
}

// Tree check and CSR form on the stack (no allocation): the same checks and
// slot order as relaysum_create.
int static_tree(int32_t n, const int32_t *edges, int32_t num_edges, StaticTopo &tp) {
    if (num_edges > 0 && !edges) return static_fail(RELAYSUM_ERR_INVALID_ARG, "edges is NULL");
    if (num_edges != n - 1) return static_fail(RELAYSUM_ERR_NOT_A_TREE, "num_edges != n - 1");
    int32_t parent[kStaticMaxWorkers];
    int32_t su[2 * (kStaticMaxWorkers - 1)], sv[2 * (kStaticMaxWorkers - 1)];
    for (int32_t i = 0; i < n; ++i) parent[i] = i;
    auto find = [&](int32_t v) {
        while (parent[v] != v) v = parent[v] = parent[parent[v]];
        return v;
    };
    int e2 = 0;
    for (int32_t e = 0; e < num_edges; ++e) {
        const int32_t u = edges[2 * e], v = edges[2 * e + 1];
        if (u < 0 || v < 0 || u >= n || v >= n || u == v)
            return static_fail(RELAYSUM_ERR_NOT_A_TREE, "edge id out of range or self loop");
        const int32_t ru = find(u), rv = find(v);
        if (ru == rv) return static_fail(RELAYSUM_ERR_NOT_A_TREE, "duplicate edge or cycle");
        parent[ru] = rv;
        su[e2] = u; sv[e2] = v; ++e2;
        su[e2] = v; sv[e2] = u; ++e2;
    }
    for (int a = 1; a < e2; ++a)   // directed edges by (source, destination)
        for (int b = a; b > 0 && (su[b - 1] > su[b] || (su[b - 1] == su[b] && sv[b - 1] > sv[b])); --b) {
            std::swap(su[b - 1], su[b]);
            std::swap(sv[b - 1], sv[b]);
        }
    tp.n = n;
    tp.e2 = e2;
    for (int32_t i = 0; i <= n; ++i) tp.row_ptr[i] = 0;
    for (int s = 0; s < e2; ++s) {
        tp.src[s] = su[s];
        tp.col[s] = sv[s];
        tp.row_ptr[su[s] + 1]++;
    }
    for (int32_t i = 0; i < n; ++i) tp.row_ptr[i + 1] += tp.row_ptr[i];
    for (int s = 0; s < e2; ++s) {
        const int32_t j = tp.col[s], i = tp.src[s];
        int r = tp.row_ptr[j];
        while (tp.col[r] != i) ++r;
        tp.rev[s] = r;
    }
    return RELAYSUM_OK;
}

uint64_t static_digest(const StaticTopo &tp) {
    uint64_t x = 1469598103934665603ull;   // FNV-1a
    auto mix = [&](int64_t v) {
        for (int b = 0; b < 8; ++b) {
            x ^= (uint64_t)((v >> (8 * b)) & 0xff);
            x *= 1099511628211ull;
        }
    };
    mix(tp.n);
    for (int32_t i = 0; i <= tp.n; ++i) mix(tp.row_ptr[i]);
    for (int s = 0; s < tp.e2; ++s) mix(tp.col[s]);
    return x;
}

size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

}  // namespace

extern "C" int relaysum_step_static(int32_t n, int64_t d, const int32_t *edges, int32_t num_edges,
                                    int64_t t, float *x, const float *g, float *mom, float lr,
                                    float beta, void *hip_stream) {
    if (n < 1 || n > kStaticMaxWorkers)
        return static_fail(RELAYSUM_ERR_INVALID_ARG, "n must be in 1..32");
    if (d < 0) return static_fail(RELAYSUM_ERR_INVALID_ARG, "d < 0");
    if (t < 0) return static_fail(RELAYSUM_ERR_INVALID_ARG, "t < 0");
    StaticTopo tp;
    int rc = static_tree(n, edges, num_edges, tp);
    if (rc != RELAYSUM_OK) return rc;
    if (d > 0) {
        if (!x || !g) return static_fail(RELAYSUM_ERR_INVALID_ARG, "x and g must not be NULL");
        if (beta != 0.0f && !mom) return static_fail(RELAYSUM_ERR_INVALID_ARG, "mom is NULL but beta != 0");
        const bool with_mom = beta != 0.0f;
        if (((uintptr_t)x | (uintptr_t)g | (with_mom ? (uintptr_t)mom : 0)) & 3)
            return static_fail(RELAYSUM_ERR_INVALID_ARG, "x, g and mom rows must be 4-byte aligned");
        const uintptr_t bytes = (uintptr_t)n * (uintptr_t)d * sizeof(float);
        const uintptr_t arr[3] = {(uintptr_t)x, (uintptr_t)g, with_mom ? (uintptr_t)mom : 0};
        for (int i = 0; i < 3; ++i)
            for (int j = i + 1; j < 3; ++j)
                if (arr[i] && arr[j] && arr[i] < arr[j] + bytes && arr[j] < arr[i] + bytes)
                    return static_fail(RELAYSUM_ERR_INVALID_ARG, "x, g and mom arrays overlap");
    }
    // Layout of the array for this tree: topology | counters | ring.
    const int e2 = tp.e2;
    // Ring tiles of 512 to 4096 floats (a handle's single-tree ring goes down
    // to 4 floats for short messages; the layout changes no result, and whole
    // 512-float tiles let the fill kernel clear a parity 16 bytes at a time).
    int shift = 9;
    while (shift < kRingShift && ((int64_t)1 << shift) < d) ++shift;
    const int64_t ring_tiles = (d + ((int64_t)1 << shift) - 1) >> shift;
    const size_t parity_floats = (size_t)ring_tiles * (size_t)e2 << shift;
    const size_t off_cnt = align256(((size_t)n + 1 + 3 * (size_t)e2) * sizeof(int32_t));
    const size_t off_ring = off_cnt + align256((2 * (size_t)e2 + n) * sizeof(int32_t));
    const size_t need = off_ring + 2 * parity_floats * sizeof(float);
    if (d > (int64_t)kStaticBytes || need > kStaticBytes) {
        char msg[160];
        std::snprintf(msg, sizeof msg, "the round needs %zu bytes of device state, the static buffer holds %zu",
                      d > (int64_t)kStaticBytes ? (size_t)-1 : need, kStaticBytes);
        return static_fail(RELAYSUM_ERR_INVALID_ARG, msg);
    }

    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return static_fail(RELAYSUM_ERR_DEVICE, "hipGetDevice failed");
    if (dev < 0 || dev >= kStaticMaxDevices) return static_fail(RELAYSUM_ERR_INVALID_ARG, "device id above 63");
    std::lock_guard<std::mutex> lock(g_static_mu);
    StaticDevice &sd = g_static[dev];
    if (!sd.base) {
        // Set-up on this device, with it current: the array's device address,
        // the device's limits, and the tile kernels' dynamic-LDS limit.
        void *p = nullptr;
        const hipError_t st = hipGetSymbolAddress(&p, HIP_SYMBOL(static_scratch));
        if (st != hipSuccess || !p) {
            (void)hipGetLastError();
            return static_fail(RELAYSUM_ERR_DEVICE, "hipGetSymbolAddress of the static buffer failed");
        }
        int v = 0;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0)
            sd.cu_count = v;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) == hipSuccess && v > 0)
            sd.lds_limit = (size_t)v;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev) == hipSuccess &&
            v > 0)
            sd.lds_cu = (size_t)v;
        for (int rule : {(int)kModelSgd, (int)kModelNesterov})
            for (int pw = 1; pw <= 2; ++pw)
                for (int nt = 0; nt < 2; ++nt)
                    for (int tail = 0; tail < 2; ++tail) {
                        const hipError_t sa = hipFuncSetAttribute((const void *)pick_tile(rule, pw, nt, tail),
                                                                  hipFuncAttributeMaxDynamicSharedMemorySize,
                                                                  (int)sd.lds_limit);
                        if (sa != hipSuccess) {
                            (void)hipGetLastError();
                            return static_fail(RELAYSUM_ERR_DEVICE, "hipFuncSetAttribute failed");
                        }
                    }
        sd.base = static_cast<unsigned char *>(p);
    }
    if (d > 0) {
        // The arrays must be n*d floats of device memory on this GPU (a kernel
        // would fault on host memory or a short buffer); the last call's
        // arrays are not queried again.
        const size_t bytes = (size_t)n * (size_t)d * sizeof(float);
        const void *arr[3] = {x, g, beta != 0.0f ? mom : nullptr};
        const char *name[3] = {"x", "g", "mom"};
        for (int i = 0; i < 3; ++i) {
            if (!arr[i] || (arr[i] == sd.checked[i] && bytes <= sd.checked_bytes)) continue;
            if (!on_device(arr[i], bytes, dev)) {
                char msg[96];
                std::snprintf(msg, sizeof msg, "%s is not n*d floats of device memory on the current GPU",
                              name[i]);
                return static_fail(RELAYSUM_ERR_INVALID_ARG, msg);
            }
        }
        for (int i = 0; i < 3; ++i) sd.checked[i] = arr[i];
        sd.checked_bytes = bytes;
    }
    const uint64_t digest = static_digest(tp);
    if (t > 0 && !(sd.run && sd.n == n && sd.d == d && sd.digest == digest && sd.next_t == t))
        return static_fail(RELAYSUM_ERR_INVALID_ARG,
                           "the static buffer of this device holds no round t-1 of this tree and d "
                           "(start a run with t = 0)");

    // Launch shape of the handle's tile kernel for this tree.
    const int waves = std::min<int>(n, kMaxWaves);
    const int pw = n <= kMaxWaves ? 1 : 2;
    const int rule = beta != 0.0f ? kModelNesterov : kModelSgd;
    const int64_t ntiles = (d + kWave * kU4 * 4 - 1) / (kWave * kU4 * 4);
    const int64_t grid = std::max<int64_t>(ntiles, 1);
    if (grid > 0x7fffffff) return static_fail(RELAYSUM_ERR_INVALID_ARG, "d too large");
    const size_t rows = beta != 0.0f ? 3 : 2;
    const bool nt = (rows * (size_t)n * (size_t)d + 2 * parity_floats) * sizeof(float) > kMallBytes / 2;
    const int per_cu = std::max(1, kMaxWaves / waves);
    const size_t cap_lds = grid >= 8 * (int64_t)sd.cu_count
                               ? std::min(sd.lds_cu / (size_t)(per_cu + 1) + 256, sd.lds_limit)
                               : 0;
    const size_t lds = std::max(tile_lds_bytes(n, e2, 4 * kU4, false), cap_lds);
    if (lds > sd.lds_limit) return static_fail(RELAYSUM_ERR_INVALID_ARG, "tree too large for LDS");
    const kernel_fn fn = pick_tile(rule, pw, nt, d % 4 != 0);

    int32_t *topo = reinterpret_cast<int32_t *>(sd.base);
    int32_t *cnt = reinterpret_cast<int32_t *>(sd.base + off_cnt);
    float *ring = reinterpret_cast<float *>(sd.base + off_ring);
    const int prev = (int)((t + 1) & 1), next = (int)(t & 1);
    RoundArgs a;
    std::memset(&a, 0, sizeof a);
    a.x = x;
    a.g = g;
    a.s1 = beta != 0.0f ? mom : nullptr;
    a.ring_prev = ring + (size_t)prev * parity_floats;
    a.ring_next = ring + (size_t)next * parity_floats;
    a.d = d;
    a.nchunks = d / 4;
    a.ntiles = ntiles;
    a.cnt_prev = cnt + (size_t)prev * e2;
    a.cnt_next = cnt + (size_t)next * e2;
    a.nbar_out = cnt + 2 * (size_t)e2;
    a.row_ptr = topo;
    a.col = topo + n + 1;
    a.rev = a.col + e2;
    a.src = a.rev + e2;
    a.n = n;
    a.e2 = e2;
    a.ring_shift = shift;
    a.ring_slots = e2;
    a.cstride = 1;
    a.lr = lr;
    a.beta1 = beta;
    a.one_m_b1 = 1.0f - beta;
    a.bc2_sqrt = 1.0f;

    hipStream_t stream = reinterpret_cast<hipStream_t>(hip_stream);
    sd.run = false;   // until this round is queued
    if (t == 0) {
        const int64_t ring_f4 = (int64_t)(parity_floats / 4);
        const unsigned pg = (unsigned)std::max<int64_t>(1, std::min<int64_t>((ring_f4 + 255) / 256, 4096));
        hipLaunchKernelGGL(relaysum_static_prepare, dim3(pg), dim3(256), 0, stream, tp, topo,
                           cnt + (size_t)prev * e2,
                           reinterpret_cast<f4_t *>(ring + (size_t)prev * parity_floats), ring_f4);
        const hipError_t st = hipGetLastError();
        if (st != hipSuccess) return static_fail(RELAYSUM_ERR_DEVICE, hipGetErrorString(st));
    }
    hipLaunchKernelGGL(fn, dim3((unsigned)grid), dim3(waves * kWave), lds, stream, a);
    const hipError_t st = hipGetLastError();
    if (st != hipSuccess) return static_fail(RELAYSUM_ERR_DEVICE, hipGetErrorString(st));
    sd.run = true;
    sd.n = n;
    sd.d = d;
    sd.digest = digest;
    sd.next_t = t + 1;
    g_static_err[0] = '\0';
    return RELAYSUM_OK;
}
