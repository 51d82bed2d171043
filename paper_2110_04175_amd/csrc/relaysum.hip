// RelaySum round on CDNA4 (gfx950): HIP kernels and the C ABI of relaysum.h.
//
// One launch performs Alg. 1 of the paper (RelaySum/Model) for every worker
// of the tree, with the Nesterov local step of Appendix D.2:
//   local step, message relay + counters, count-corrected average.
//
// The round streams every model row, gradient row, momentum row and message
// row once; it does a few adds per float, so it is bound by HBM bandwidth
// (no contraction, no MFMA).  Layout in HBM:
//   x, g, mom           caller-owned float[n][d], row stride d
//   ring                float[2][ceil(d/512)][2E][512]: parity t&1 receives
//                       the messages of round t while parity (t-1)&1 holds
//                       those of round t-1.  The ring is tile-major: the 512
//                       coordinates [512k, 512k+512) of all 2E messages are
//                       one contiguous block, so the messages a workgroup
//                       streams for its tile are adjacent in HBM instead of
//                       2E rows d floats apart (5.19 -> 5.47 TB/s in a
//                       probe of this access pattern on MI355X)
//   counts              int32[2][2E] double-buffered like the ring, nbar[n]
//   tree                CSR: row_ptr[n+1]; slots row_ptr[i]..row_ptr[i+1]-1
//                       are the directed edges i->col[s], col ascending;
//                       rev[s] is the slot of the reverse edge; src[s] = i
//
// Tile kernel (trees up to a few hundred workers).  Workgroup b owns tile b:
// the same 64*U*C consecutive coordinates of every row (2048 floats on the
// 128-bit path, U = 2 float4 per lane; 64 floats on the 32-bit path).  Each
// wave owns whole workers (worker i belongs to wave i mod W).  Phase 1: a
// wave streams x_i, g_i, mom_i and the previous messages into i, forms the
// half-step xh_i (kept in registers), writes mom_i and the messages i->j to
// HBM and to an LDS tile [2E][64*U*C].  After a barrier, phase 2 forms each
// average from xh_i and the LDS copies of the new messages into i and writes
// x_i.  New messages are read back from LDS, never from HBM, so every HBM
// byte of the round is touched exactly once; all HBM accesses are
// non-temporal, as nothing is reused within a round.  Every workgroup first
// relays the (few) integer counters into LDS itself, so no grid-wide
// synchronisation is needed; workgroup 0 also publishes them.
//
// Two-pass path (larger trees, whose message tile does not fit in LDS): one
// small launch relays the counters, one writes xh into x together with the
// new messages, one forms the averages from x and the new messages.
//
// Arithmetic: one IEEE binary32 rounding per operation, contraction off, sums
// start from xh_i and add neighbours in ascending id, the average is a
// correctly rounded division.  Results do not depend on the access width,
// the tile or the grid.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstring>
#include <string>
#include <vector>

#include "relaysum.h"

#pragma clang fp contract(off)

namespace {

constexpr int kWave = 64;
constexpr int kMaxWaves = 16;       // 1024-thread workgroups
constexpr int kMaxDegInRegs = 4;    // previous messages into a worker kept in VGPRs (128-bit path)
constexpr int kMaxDegInRegs32 = 8;  // the same on the 32-bit path
constexpr int64_t kRingTile = 512;  // floats per message per ring tile (2 KB)

// A lane's share of one row within a tile: U chunks of C floats (C = 4 for
// 128-bit accesses, C = 1 otherwise).  Chunk u of lane l lies at float offset
// (u*64 + l)*C from the tile start, so every wave-wide access covers 64*C
// contiguous floats (1 KB when C = 4).
template <int U, int C>
struct lanev {
    float v[U][C];
};

typedef float f4_t __attribute__((ext_vector_type(4)));

// Every model, gradient, momentum and message row is touched once per round,
// so loads and stores are non-temporal (streamed past the caches).
template <int C>
__device__ __forceinline__ void load_chunk(const float *p, float (&r)[C]) {
    if constexpr (C == 4) {
        const f4_t t = __builtin_nontemporal_load(reinterpret_cast<const f4_t *>(p));
        r[0] = t.x; r[1] = t.y; r[2] = t.z; r[3] = t.w;
    } else {
#pragma unroll
        for (int k = 0; k < C; ++k) r[k] = __builtin_nontemporal_load(p + k);
    }
}

template <int C>
__device__ __forceinline__ void store_chunk(float *p, const float (&a)[C]) {
    if constexpr (C == 4) {
        const f4_t t = {a[0], a[1], a[2], a[3]};
        __builtin_nontemporal_store(t, reinterpret_cast<f4_t *>(p));
    } else {
#pragma unroll
        for (int k = 0; k < C; ++k) __builtin_nontemporal_store(a[k], p + k);
    }
}

// Load a lane's chunks of one row; `row` points at the tile start of the row.
template <int U, int C>
__device__ __forceinline__ lanev<U, C> load_lane(const float *row, int lane, const bool (&ok)[U]) {
    lanev<U, C> r;
#pragma unroll
    for (int u = 0; u < U; ++u) {
        if (ok[u]) {
            load_chunk<C>(row + (u * 64 + lane) * C, r.v[u]);
        } else {
#pragma unroll
            for (int k = 0; k < C; ++k) r.v[u][k] = 0.0f;
        }
    }
    return r;
}

template <int U, int C>
__device__ __forceinline__ void store_lane(float *row, int lane, const bool (&ok)[U],
                                           const lanev<U, C> &a) {
#pragma unroll
    for (int u = 0; u < U; ++u)
        if (ok[u]) store_chunk<C>(row + (u * 64 + lane) * C, a.v[u]);
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

// Local half-step (Alg. 1 line 3; Appendix D.2), one IEEE operation per line.
// With momentum: b <- beta*b + g; xh = x - lr*(g + beta*b).
template <int U, int C, bool MOM>
__device__ __forceinline__ lanev<U, C> half_step(const lanev<U, C> &x, const lanev<U, C> &g,
                                                 lanev<U, C> &b, float lr, float beta) {
    lanev<U, C> xh;
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
        for (int k = 0; k < C; ++k) {
            if constexpr (MOM) {
                const float p = beta * b.v[u][k];
                const float bn = p + g.v[u][k];
                b.v[u][k] = bn;
                const float q = beta * bn;
                const float w = g.v[u][k] + q;
                const float s = lr * w;
                xh.v[u][k] = x.v[u][k] - s;
            } else {
                const float s = lr * g.v[u][k];
                xh.v[u][k] = x.v[u][k] - s;
            }
        }
    return xh;
}

struct RoundArgs {
    float *x;
    const float *g;
    float *mom;
    const float *ring_prev;   // messages of round t-1, [ceil(d/512)][2E][512]
    float *ring_next;         // messages of round t
    int64_t d;                // floats per model row
    int64_t nchunks;          // d / C (C-float chunks per row)
    int64_t ntiles;           // tiles per row (64*U chunks each)
    const int32_t *cnt_prev;  // c^{(t-1)} per slot
    int32_t *cnt_next;        // c^{(t)} per slot
    int32_t *nbar_out;        // nbar_i of round t
    const int32_t *row_ptr;
    const int32_t *col;
    const int32_t *rev;
    const int32_t *src;
    int32_t n;
    int32_t e2;
    float lr;
    float beta;
};

__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

// Address of message `slot` at coordinate c in a tile-major ring parity.
// Kernel tiles and chunks never straddle a 512-float ring tile.
__device__ __forceinline__ int64_t ring_off(int e2, int slot, int64_t c) {
    return ((c / kRingTile) * e2 + slot) * kRingTile + (c % kRingTile);
}

// Counter relay of Alg. 1 into LDS: c_{i->j} = 1 + sum_{k in N_i\j} c_{k->i}
// over the previous round's counters, then nbar_i = 1 + sum_j c_{j->i}.
__device__ void relay_counts(const RoundArgs &a, int32_t *s_cnt, int32_t *s_nbar) {
    for (int s = threadIdx.x; s < a.e2; s += blockDim.x) {
        const int i = a.src[s], j = a.col[s];
        int c = 1;
        for (int q = a.row_ptr[i]; q < a.row_ptr[i + 1]; ++q)
            if (a.col[q] != j) c += a.cnt_prev[a.rev[q]];
        s_cnt[s] = c;
    }
    __syncthreads();
    for (int i = threadIdx.x; i < a.n; i += blockDim.x) {
        int nb = 1;
        for (int q = a.row_ptr[i]; q < a.row_ptr[i + 1]; ++q) nb += s_cnt[a.rev[q]];
        s_nbar[i] = nb;
    }
    __syncthreads();
}

// Messages out of worker i (Alg. 1): for each neighbour j (slot s0+q),
// m_{i->j} = xh_i + sum over the other in-edges b != q, ascending, of the
// previous round's m_{k->i}.  `o` holds those previous messages when the
// degree is at most MD; larger degrees re-read them from HBM (cache hits).
// Each message goes to the ring (HBM) and to the LDS tile.
template <int U, int C, int MD>
__device__ __forceinline__ void emit_messages(const RoundArgs &a, float *s_msg, int slot_floats,
                                              int lane, const bool (&ok)[U], int64_t base, int s0,
                                              int deg, const lanev<U, C> &xh,
                                              const lanev<U, C> (&o)[MD]) {
    if (deg <= MD) {
#pragma unroll
        for (int q = 0; q < MD; ++q) {
            if (q < deg) {
                lanev<U, C> m = xh;
#pragma unroll
                for (int b = 0; b < MD; ++b)
                    if (b < deg && b != q) m = add_lane<U, C>(m, o[b]);
                store_lane<U, C>(a.ring_next + ring_off(a.e2, (s0 + q), base), lane, ok, m);
                lds_put<U, C>(s_msg + (s0 + q) * slot_floats, lane, m);
            }
        }
    } else {
        for (int q = 0; q < deg; ++q) {
            lanev<U, C> m = xh;
            for (int b = 0; b < deg; ++b) {
                if (b == q) continue;
                const int in_slot = uniform(a.rev[s0 + b]);
                m = add_lane<U, C>(
                    m, load_lane<U, C>(a.ring_prev + ring_off(a.e2, in_slot, base), lane, ok));
            }
            store_lane<U, C>(a.ring_next + ring_off(a.e2, (s0 + q), base), lane, ok, m);
            lds_put<U, C>(s_msg + (s0 + q) * slot_floats, lane, m);
        }
    }
}

// Tile kernel: workgroup b owns tile b, the 64*U*C consecutive coordinates
// starting at b*64*U*C, for every row.
template <int U, int C, int PW, bool MOM>
__global__ void __launch_bounds__(1024) relaysum_tile_kernel(RoundArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    int32_t *s_cnt = reinterpret_cast<int32_t *>(smem);
    int32_t *s_nbar = s_cnt + a.e2;
    const int hdr = ((a.e2 + a.n) * 4 + 15) & ~15;
    float *s_msg = reinterpret_cast<float *>(smem + hdr);   // [2E][U][64][C]
    constexpr int kSlot = 64 * U * C;                        // floats per LDS message slot

    relay_counts(a, s_cnt, s_nbar);
    if (blockIdx.x == 0) {
        for (int s = threadIdx.x; s < a.e2; s += blockDim.x) a.cnt_next[s] = s_cnt[s];
        for (int i = threadIdx.x; i < a.n; i += blockDim.x) a.nbar_out[i] = s_nbar[i];
    }

    const int lane = threadIdx.x & (kWave - 1);
    const int wave = uniform(threadIdx.x >> 6);
    const int W = blockDim.x >> 6;
    const int64_t tile = blockIdx.x;
    const int64_t base = tile * kSlot;   // float offset of the tile in every row
    bool ok[U];
#pragma unroll
    for (int u = 0; u < U; ++u) ok[u] = (tile * 64 * U + u * 64 + lane) < a.nchunks;

    lanev<U, C> xh[PW];
    // Phase 1: half-steps, momentum, outgoing messages.
    if constexpr (C == 4) {
        // 128-bit path (one or two workers per wave): all loads of a worker
        // are issued before any of its arithmetic.
#pragma unroll
        for (int p = 0; p < PW; ++p) {
            const int i = wave + p * W;
            if (i >= a.n) break;
            const int64_t row = (int64_t)i * a.d + base;
            const lanev<U, C> xv = load_lane<U, C>(a.x + row, lane, ok);
            const lanev<U, C> gv = load_lane<U, C>(a.g + row, lane, ok);
            lanev<U, C> bv = zero_lane<U, C>();
            if constexpr (MOM) bv = load_lane<U, C>(a.mom + row, lane, ok);
            const int s0 = uniform(a.row_ptr[i]);
            const int deg = uniform(a.row_ptr[i + 1]) - s0;
            lanev<U, C> o[kMaxDegInRegs];
            if (deg <= kMaxDegInRegs) {
#pragma unroll
                for (int b = 0; b < kMaxDegInRegs; ++b) {
                    if (b < deg) {
                        const int in_slot = uniform(a.rev[s0 + b]);
                        o[b] = load_lane<U, C>(a.ring_prev + ring_off(a.e2, in_slot, base), lane, ok);
                    }
                }
            }
            xh[p] = half_step<U, C, MOM>(xv, gv, bv, a.lr, a.beta);
            if constexpr (MOM) store_lane<U, C>(a.mom + row, lane, ok, bv);
            emit_messages<U, C, kMaxDegInRegs>(a, s_msg, kSlot, lane, ok, base, s0, deg, xh[p], o);
        }
    } else {
        // 32-bit path, up to 32 workers per wave: loads are issued for a group
        // of workers at a time so that many rows are in flight per wave.
        constexpr int GA = PW < 8 ? PW : 8;   // workers per group, half-steps
        constexpr int GB = PW < 4 ? PW : 4;   // workers per group, messages
#pragma unroll
        for (int p0 = 0; p0 < PW; p0 += GA) {
            lanev<U, C> xv[GA], gv[GA], bv[GA];
#pragma unroll
            for (int p = 0; p < GA; ++p) {
                const int i = wave + (p0 + p) * W;
                if (i < a.n) {
                    const int64_t row = (int64_t)i * a.d + base;
                    xv[p] = load_lane<U, C>(a.x + row, lane, ok);
                    gv[p] = load_lane<U, C>(a.g + row, lane, ok);
                    bv[p] = zero_lane<U, C>();
                    if constexpr (MOM) bv[p] = load_lane<U, C>(a.mom + row, lane, ok);
                }
            }
#pragma unroll
            for (int p = 0; p < GA; ++p) {
                const int i = wave + (p0 + p) * W;
                if (i < a.n) {
                    xh[p0 + p] = half_step<U, C, MOM>(xv[p], gv[p], bv[p], a.lr, a.beta);
                    if constexpr (MOM) store_lane<U, C>(a.mom + (int64_t)i * a.d + base, lane, ok, bv[p]);
                }
            }
        }
        constexpr int MD = kMaxDegInRegs32;
#pragma unroll
        for (int p0 = 0; p0 < PW; p0 += GB) {
            lanev<U, C> o[GB][MD];
            int s0[GB], deg[GB];
#pragma unroll
            for (int p = 0; p < GB; ++p) {
                const int i = wave + (p0 + p) * W;
                s0[p] = 0;
                deg[p] = 0;
                if (i < a.n) {
                    s0[p] = uniform(a.row_ptr[i]);
                    deg[p] = uniform(a.row_ptr[i + 1]) - s0[p];
                }
                if (deg[p] <= MD) {
#pragma unroll
                    for (int b = 0; b < MD; ++b) {
                        if (b < deg[p]) {
                            const int in_slot = uniform(a.rev[s0[p] + b]);
                            o[p][b] = load_lane<U, C>(a.ring_prev + ring_off(a.e2, in_slot, base), lane, ok);
                        }
                    }
                }
            }
#pragma unroll
            for (int p = 0; p < GB; ++p)
                emit_messages<U, C, MD>(a, s_msg, kSlot, lane, ok, base, s0[p], deg[p], xh[p0 + p], o[p]);
        }
    }
    __syncthreads();
    // Phase 2: count-corrected averages.
#pragma unroll
    for (int p = 0; p < PW; ++p) {
        const int i = wave + p * W;
        if (i >= a.n) break;
        const int s0 = uniform(a.row_ptr[i]);
        const int deg = uniform(a.row_ptr[i + 1]) - s0;
        lanev<U, C> acc = xh[p];
        for (int q = 0; q < deg; ++q) {
            const int in_slot = uniform(a.rev[s0 + q]);
            acc = add_lane<U, C>(acc, lds_get<U, C>(s_msg + in_slot * kSlot, lane));
        }
        const float nb = (float)s_nbar[i];
        lanev<U, C> xn;
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int k = 0; k < C; ++k) xn.v[u][k] = acc.v[u][k] / nb;
        store_lane<U, C>(a.x + (int64_t)i * a.d + base, lane, ok, xn);
    }
}

// ---- two-pass path --------------------------------------------------------

__global__ void __launch_bounds__(1024) relaysum_count_kernel(RoundArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    int32_t *s_cnt = reinterpret_cast<int32_t *>(smem);
    int32_t *s_nbar = s_cnt + a.e2;
    relay_counts(a, s_cnt, s_nbar);
    for (int s = threadIdx.x; s < a.e2; s += blockDim.x) a.cnt_next[s] = s_cnt[s];
    for (int i = threadIdx.x; i < a.n; i += blockDim.x) a.nbar_out[i] = s_nbar[i];
}

// Half-step and outgoing messages of worker blockIdx.y (grid-strided); the
// half-step is left in x for the averaging pass.  Each thread handles one
// C-float chunk per iteration.
template <int C, bool MOM>
__global__ void __launch_bounds__(256) relaysum_pass_a(RoundArgs a) {
    const bool ok[1] = {true};
    constexpr int MD = kMaxDegInRegs32;
    for (int i = blockIdx.y; i < a.n; i += gridDim.y) {
        const int s0 = a.row_ptr[i];
        const int deg = a.row_ptr[i + 1] - s0;
        for (int64_t chunk = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; chunk < a.nchunks;
             chunk += (int64_t)gridDim.x * blockDim.x) {
            const int64_t off = chunk * C;
            const int64_t row = (int64_t)i * a.d + off;
            const lanev<1, C> xv = load_lane<1, C>(a.x + row, 0, ok);
            const lanev<1, C> gv = load_lane<1, C>(a.g + row, 0, ok);
            lanev<1, C> bv = zero_lane<1, C>();
            if constexpr (MOM) bv = load_lane<1, C>(a.mom + row, 0, ok);
            lanev<1, C> o[MD];
            if (deg <= MD) {
#pragma unroll
                for (int b = 0; b < MD; ++b)
                    if (b < deg)
                        o[b] = load_lane<1, C>(a.ring_prev + ring_off(a.e2, a.rev[s0 + b], off), 0, ok);
            }
            const lanev<1, C> xh = half_step<1, C, MOM>(xv, gv, bv, a.lr, a.beta);
            if constexpr (MOM) store_lane<1, C>(a.mom + row, 0, ok, bv);
            if (deg <= MD) {
#pragma unroll
                for (int q = 0; q < MD; ++q) {
                    if (q < deg) {
                        lanev<1, C> m = xh;
#pragma unroll
                        for (int b = 0; b < MD; ++b)
                            if (b < deg && b != q) m = add_lane<1, C>(m, o[b]);
                        store_lane<1, C>(a.ring_next + ring_off(a.e2, (s0 + q), off), 0, ok, m);
                    }
                }
            } else {
                for (int q = 0; q < deg; ++q) {
                    lanev<1, C> m = xh;
                    for (int b = 0; b < deg; ++b) {
                        if (b == q) continue;
                        m = add_lane<1, C>(m, load_lane<1, C>(a.ring_prev + ring_off(a.e2, a.rev[s0 + b], off), 0, ok));
                    }
                    store_lane<1, C>(a.ring_next + ring_off(a.e2, (s0 + q), off), 0, ok, m);
                }
            }
            store_lane<1, C>(a.x + row, 0, ok, xh);
        }
    }
}

template <int C>
__global__ void __launch_bounds__(256) relaysum_pass_b(RoundArgs a) {
    const bool ok[1] = {true};
    for (int i = blockIdx.y; i < a.n; i += gridDim.y) {
        const int s0 = a.row_ptr[i];
        const int deg = a.row_ptr[i + 1] - s0;
        const float nb = (float)a.nbar_out[i];
        for (int64_t chunk = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; chunk < a.nchunks;
             chunk += (int64_t)gridDim.x * blockDim.x) {
            const int64_t off = chunk * C;
            const int64_t row = (int64_t)i * a.d + off;
            lanev<1, C> acc = load_lane<1, C>(a.x + row, 0, ok);
            for (int q = 0; q < deg; ++q)
                acc = add_lane<1, C>(acc, load_lane<1, C>(a.ring_next + ring_off(a.e2, a.rev[s0 + q], off), 0, ok));
            lanev<1, C> xn;
#pragma unroll
            for (int k = 0; k < C; ++k) xn.v[0][k] = acc.v[0][k] / nb;
            store_lane<1, C>(a.x + row, 0, ok, xn);
        }
    }
}

// ---- host side --------------------------------------------------------------

typedef void (*tile_fn)(RoundArgs);

// 128-bit path: each lane streams U = 2 float4 chunks per row and tile (a
// 2 KB tile row per wave), at most two workers per wave.  32-bit path (rows
// not 16-byte aligned): one float per lane.
constexpr int kU4 = 2;

template <bool MOM>
tile_fn pick_tile_v4(int pw) {
    switch (pw) {
        case 1: return relaysum_tile_kernel<kU4, 4, 1, MOM>;
        case 2: return relaysum_tile_kernel<kU4, 4, 2, MOM>;
        default: return nullptr;
    }
}

template <bool MOM>
tile_fn pick_tile_v1(int pw) {
    switch (pw) {
        case 1: return relaysum_tile_kernel<1, 1, 1, MOM>;
        case 2: return relaysum_tile_kernel<1, 1, 2, MOM>;
        default: return nullptr;
    }
}

// LDS of the tile kernel: counters and nbar, then the [2E][64 * floats_per_lane] message tile.
size_t tile_lds_bytes(int n, int e2, int floats_per_lane) {
    const size_t hdr = (((size_t)e2 + n) * 4 + 15) & ~(size_t)15;
    return hdr + (size_t)e2 * kWave * floats_per_lane * sizeof(float);
}

}  // namespace

struct relaysum_s {
    int32_t n = 0;
    int64_t d = 0;
    int32_t e2 = 0;
    std::vector<int32_t> row_ptr, col, rev, src;
    int32_t *d_topo = nullptr;   // row_ptr[n+1] | col[e2] | rev[e2] | src[e2]
    int32_t *d_counts = nullptr; // cnt[2][e2] | nbar[n]
    float *ring = nullptr;       // [2][ring_tiles][e2][512]
    int64_t ring_tiles = 0;      // ceil(d / 512)
    int64_t t = 0;
    hipStream_t stream = nullptr;
    int device = 0;
    int cu_count = 256;
    int waves = 1;               // W: waves per workgroup of the tile kernel
    int pw = 1;                  // workers per wave (power of two)
    int tile_v = 0;              // 4: 128-bit tile kernel, 1: 32-bit tile kernel, 0: two-pass
    size_t lds_limit = 64 * 1024;   // LDS one workgroup may use
    size_t lds_cu = 160 * 1024;     // LDS of one CU (gfx950)
    struct Launch {
        tile_fn fn = nullptr;
        size_t lds = 0;
    } launch[2][2];              // [128-bit][momentum], filled on first use
    std::string err;
};

// Floats in one parity of the tile-major message ring.
static size_t ring_parity_floats(const relaysum_t *h) {
    return (size_t)h->ring_tiles * (size_t)h->e2 * kRingTile;
}

static int fail(relaysum_t *h, int code, const std::string &msg) {
    if (h) h->err = msg;
    return code;
}

static int hip_fail(relaysum_t *h, hipError_t e, const char *what) {
    return fail(h, RELAYSUM_ERR_DEVICE, std::string(what) + ": " + hipGetErrorString(e));
}

static void release(relaysum_t *h) {
    if (!h) return;
    if (h->ring) (void)hipFree(h->ring);
    if (h->d_counts) (void)hipFree(h->d_counts);
    if (h->d_topo) (void)hipFree(h->d_topo);
    delete h;
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

const char *relaysum_last_error(const relaysum_t *h) { return h ? h->err.c_str() : ""; }

int relaysum_create(int32_t n, int64_t d, const int32_t *edges, int32_t num_edges,
                    relaysum_t **out) {
    if (!out) return RELAYSUM_ERR_INVALID_ARG;
    *out = nullptr;
    if (n < 1 || d < 0) return RELAYSUM_ERR_INVALID_ARG;
    if (num_edges > 0 && !edges) return RELAYSUM_ERR_INVALID_ARG;
    if (num_edges != n - 1) return RELAYSUM_ERR_NOT_A_TREE;

    // Validate: ids in range, no self loops, no duplicates, connected.
    std::vector<std::pair<int32_t, int32_t>> dir;
    dir.reserve(2 * (size_t)num_edges);
    std::vector<int32_t> parent(n);
    for (int32_t i = 0; i < n; ++i) parent[i] = i;
    auto find = [&](int32_t v) {
        while (parent[v] != v) { parent[v] = parent[parent[v]]; v = parent[v]; }
        return v;
    };
    for (int32_t e = 0; e < num_edges; ++e) {
        const int32_t u = edges[2 * e], v = edges[2 * e + 1];
        if (u < 0 || v < 0 || u >= n || v >= n || u == v) return RELAYSUM_ERR_NOT_A_TREE;
        const int32_t ru = find(u), rv = find(v);
        if (ru == rv) return RELAYSUM_ERR_NOT_A_TREE;   // duplicate edge or cycle
        parent[ru] = rv;
        dir.emplace_back(u, v);
        dir.emplace_back(v, u);
    }
    // n-1 edges without a cycle connect all n workers.
    std::sort(dir.begin(), dir.end());

    relaysum_t *h = new (std::nothrow) relaysum_s();
    if (!h) return RELAYSUM_ERR_OUT_OF_MEMORY;
    h->n = n;
    h->d = d;
    h->e2 = (int32_t)dir.size();
    h->row_ptr.assign(n + 1, 0);
    h->col.resize(h->e2);
    h->src.resize(h->e2);
    h->rev.resize(h->e2);
    for (int32_t s = 0; s < h->e2; ++s) {
        h->src[s] = dir[s].first;
        h->col[s] = dir[s].second;
        h->row_ptr[dir[s].first + 1]++;
    }
    for (int32_t i = 0; i < n; ++i) h->row_ptr[i + 1] += h->row_ptr[i];
    for (int32_t s = 0; s < h->e2; ++s) {
        const int32_t j = h->col[s], i = h->src[s];
        const auto b = h->col.begin() + h->row_ptr[j], e = h->col.begin() + h->row_ptr[j + 1];
        h->rev[s] = (int32_t)(std::lower_bound(b, e, i) - h->col.begin());
    }

    hipError_t st = hipGetDevice(&h->device);
    if (st != hipSuccess) { release(h); return RELAYSUM_ERR_DEVICE; }
    int cus = 0, lds_max = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, h->device) == hipSuccess &&
        cus > 0)
        h->cu_count = cus;
    if (hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, h->device) ==
            hipSuccess && lds_max > 0)
        h->lds_limit = (size_t)lds_max;
    int lds_cu = 0;
    if (hipDeviceGetAttribute(&lds_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor,
                              h->device) == hipSuccess && lds_cu > 0)
        h->lds_cu = (size_t)lds_cu;

    // Tile plan: W waves per workgroup, pw workers per wave, V floats per lane.
    h->waves = std::min<int>(n, kMaxWaves);
    int pw = 1;
    while (pw * h->waves < n) pw *= 2;
    h->pw = pw;
    // Trees of up to 32 workers use the tile kernel.  Wider trees use the
    // two-pass path: their [2E][64]-float message tile fills LDS, leaving one
    // workgroup per CU and 256-byte row segments, and on the 256-worker random
    // tree that ran at 4.24 ms per round against 2.38 ms for the two-pass path
    // (which moves 1.44x the bytes but streams them at full rate).
    if (pw <= 2) {
        if (tile_lds_bytes(n, h->e2, 4 * kU4) <= h->lds_limit) h->tile_v = 4;
        else if (tile_lds_bytes(n, h->e2, 1) <= h->lds_limit) h->tile_v = 1;
    }

    const size_t topo_ints = (size_t)(n + 1) + 3 * (size_t)h->e2;
    if (hipMalloc(&h->d_topo, topo_ints * sizeof(int32_t)) != hipSuccess ||
        hipMalloc(&h->d_counts, (2 * (size_t)h->e2 + n) * sizeof(int32_t)) != hipSuccess) {
        release(h);
        return RELAYSUM_ERR_OUT_OF_MEMORY;
    }
    h->ring_tiles = (d + kRingTile - 1) / kRingTile;
    if (h->e2 > 0 && d > 0) {
        const size_t bytes = 2 * ring_parity_floats(h) * sizeof(float);
        if (hipMalloc(&h->ring, bytes) != hipSuccess) {
            (void)hipGetLastError();
            release(h);
            return RELAYSUM_ERR_OUT_OF_MEMORY;
        }
    }
    std::vector<int32_t> topo;
    topo.reserve(topo_ints);
    topo.insert(topo.end(), h->row_ptr.begin(), h->row_ptr.end());
    topo.insert(topo.end(), h->col.begin(), h->col.end());
    topo.insert(topo.end(), h->rev.begin(), h->rev.end());
    topo.insert(topo.end(), h->src.begin(), h->src.end());
    st = hipMemcpy(h->d_topo, topo.data(), topo_ints * sizeof(int32_t), hipMemcpyHostToDevice);
    if (st != hipSuccess) { release(h); return RELAYSUM_ERR_DEVICE; }
    if (relaysum_reset(h) != RELAYSUM_OK || hipStreamSynchronize(h->stream) != hipSuccess) {
        release(h);
        return RELAYSUM_ERR_DEVICE;
    }
    *out = h;
    return RELAYSUM_OK;
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
    hipError_t st = hipMemsetAsync(h->d_counts, 0, (2 * (size_t)h->e2 + h->n) * sizeof(int32_t),
                                   h->stream);
    if (st == hipSuccess && h->ring)
        st = hipMemsetAsync(h->ring, 0,
                            2 * ring_parity_floats(h) * sizeof(float), h->stream);
    if (st != hipSuccess) return hip_fail(h, st, "reset");
    h->t = 0;
    return RELAYSUM_OK;
}

int relaysum_round(const relaysum_t *h, int64_t *t) {
    if (!h || !t) return RELAYSUM_ERR_INVALID_ARG;
    *t = h->t;
    return RELAYSUM_OK;
}

int relaysum_num_directed_edges(const relaysum_t *h, int32_t *count) {
    if (!h || !count) return RELAYSUM_ERR_INVALID_ARG;
    *count = h->e2;
    return RELAYSUM_OK;
}

int relaysum_directed_edge(const relaysum_t *h, int32_t slot, int32_t *src, int32_t *dst) {
    if (!h || slot < 0 || slot >= h->e2) return RELAYSUM_ERR_INVALID_ARG;
    if (src) *src = h->src[slot];
    if (dst) *dst = h->col[slot];
    return RELAYSUM_OK;
}

int relaysum_step(relaysum_t *h, float *x, const float *g, float *mom, float lr, float beta) {
    if (!h) return RELAYSUM_ERR_INVALID_ARG;
    const bool use_mom = beta != 0.0f;
    if (h->d > 0) {
        if (!x || !g) return fail(h, RELAYSUM_ERR_INVALID_ARG, "x and g must not be NULL");
        if (use_mom && !mom) return fail(h, RELAYSUM_ERR_INVALID_ARG, "mom is NULL but beta != 0");
        const uintptr_t bits = (uintptr_t)x | (uintptr_t)g | (use_mom ? (uintptr_t)mom : 0);
        if (bits & 3) return fail(h, RELAYSUM_ERR_INVALID_ARG, "x, g, mom must be 4-byte aligned");
    }
    const int prev = (int)((h->t + 1) & 1), next = (int)(h->t & 1);
    RoundArgs a;
    a.x = x;
    a.g = g;
    a.mom = use_mom ? mom : nullptr;
    a.ring_prev = h->ring ? h->ring + (size_t)prev * ring_parity_floats(h) : nullptr;
    a.ring_next = h->ring ? h->ring + (size_t)next * ring_parity_floats(h) : nullptr;
    a.d = h->d;
    a.cnt_prev = h->d_counts + (size_t)prev * h->e2;
    a.cnt_next = h->d_counts + (size_t)next * h->e2;
    a.nbar_out = h->d_counts + 2 * (size_t)h->e2;
    a.row_ptr = h->d_topo;
    a.col = h->d_topo + h->n + 1;
    a.rev = a.col + h->e2;
    a.src = a.rev + h->e2;
    a.n = h->n;
    a.e2 = h->e2;
    a.lr = lr;
    a.beta = beta;

    const uintptr_t bits16 = (uintptr_t)x | (uintptr_t)g | (use_mom ? (uintptr_t)mom : 0);
    const bool vec4 = (h->d % 4 == 0) && (bits16 & 15) == 0;

    if (h->tile_v) {
        const int C = (h->tile_v == 4 && vec4) ? 4 : 1;
        const int U = C == 4 ? kU4 : 1;
        a.nchunks = h->d / C;
        a.ntiles = (a.nchunks + kWave * U - 1) / (kWave * U);
        const int threads = h->waves * kWave;
        relaysum_s::Launch &L = h->launch[C == 4][use_mom];
        if (!L.fn) {
            tile_fn fn = C == 4 ? (use_mom ? pick_tile_v4<true>(h->pw) : pick_tile_v4<false>(h->pw))
                                : (use_mom ? pick_tile_v1<true>(h->pw) : pick_tile_v1<false>(h->pw));
            if (!fn) return fail(h, RELAYSUM_ERR_INVALID_ARG, "no tile kernel for this tree");
            // Residency cap of 16 waves per CU: the launch reserves enough LDS
            // that at most 16/W workgroups fit on a CU.  On the 16-worker chain
            // two co-resident 16-wave workgroups streamed 3-4% slower than one
            // (more concurrent DRAM streams per CU for the same bytes in flight).
            const int per_cu = std::max(1, kMaxWaves / h->waves);
            const size_t lds = std::max(tile_lds_bytes(h->n, h->e2, U * C),
                                        std::min(h->lds_cu / (size_t)(per_cu + 1) + 256, h->lds_limit));
            hipError_t st = hipFuncSetAttribute((const void *)fn,
                                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
            if (st != hipSuccess) return hip_fail(h, st, "hipFuncSetAttribute");
            L.fn = fn;
            L.lds = lds;
        }
        // One workgroup per tile (d == 0: one workgroup still relays the counters).
        const int64_t grid = std::max<int64_t>(a.ntiles, 1);
        if (grid > 0x7fffffff) return fail(h, RELAYSUM_ERR_INVALID_ARG, "d too large");
        hipLaunchKernelGGL(L.fn, dim3((unsigned)grid), dim3(threads), L.lds, h->stream, a);
        hipError_t st = hipGetLastError();
        if (st != hipSuccess) return hip_fail(h, st, "tile kernel launch");
    } else {
        const int V = vec4 ? 4 : 1;
        a.nchunks = h->d / V;
        a.ntiles = 0;
        const size_t lds = (((size_t)h->e2 + h->n) * 4 + 15) & ~(size_t)15;
        if (lds > h->lds_limit) return fail(h, RELAYSUM_ERR_INVALID_ARG, "tree too large");
        hipError_t st = hipFuncSetAttribute((const void *)relaysum_count_kernel,
                                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (st != hipSuccess) return hip_fail(h, st, "hipFuncSetAttribute");
        hipLaunchKernelGGL(relaysum_count_kernel, dim3(1), dim3(1024), lds, h->stream, a);
        if (a.nchunks > 0) {
            const int64_t want = (a.nchunks + 255) / 256;
            const unsigned gx = (unsigned)std::min<int64_t>(want, 1024);
            const unsigned gy = (unsigned)std::min<int64_t>(h->n, 65535);
            if (V == 4) {
                if (use_mom) hipLaunchKernelGGL((relaysum_pass_a<4, true>), dim3(gx, gy), dim3(256), 0, h->stream, a);
                else hipLaunchKernelGGL((relaysum_pass_a<4, false>), dim3(gx, gy), dim3(256), 0, h->stream, a);
                hipLaunchKernelGGL((relaysum_pass_b<4>), dim3(gx, gy), dim3(256), 0, h->stream, a);
            } else {
                if (use_mom) hipLaunchKernelGGL((relaysum_pass_a<1, true>), dim3(gx, gy), dim3(256), 0, h->stream, a);
                else hipLaunchKernelGGL((relaysum_pass_a<1, false>), dim3(gx, gy), dim3(256), 0, h->stream, a);
                hipLaunchKernelGGL((relaysum_pass_b<1>), dim3(gx, gy), dim3(256), 0, h->stream, a);
            }
        }
        st = hipGetLastError();
        if (st != hipSuccess) return hip_fail(h, st, "two-pass launch");
    }
    h->t += 1;
    return RELAYSUM_OK;
}

int relaysum_get_counts(relaysum_t *h, int32_t *nbar_host, int32_t *edge_counts_host) {
    if (!h) return RELAYSUM_ERR_INVALID_ARG;
    const int last = (int)((h->t + 1) & 1);   // slot written by round t-1
    hipError_t st = hipSuccess;
    if (edge_counts_host && h->e2 > 0)
        st = hipMemcpyAsync(edge_counts_host, h->d_counts + (size_t)last * h->e2,
                            h->e2 * sizeof(int32_t), hipMemcpyDeviceToHost, h->stream);
    if (st == hipSuccess && nbar_host)
        st = hipMemcpyAsync(nbar_host, h->d_counts + 2 * (size_t)h->e2, h->n * sizeof(int32_t),
                            hipMemcpyDeviceToHost, h->stream);
    if (st == hipSuccess) st = hipStreamSynchronize(h->stream);
    return st == hipSuccess ? RELAYSUM_OK : hip_fail(h, st, "get_counts");
}

int relaysum_get_message(relaysum_t *h, int32_t slot, float *dst_host) {
    if (!h || !dst_host || slot < 0 || slot >= h->e2) return RELAYSUM_ERR_INVALID_ARG;
    if (h->d == 0) return RELAYSUM_OK;
    const int last = (int)((h->t + 1) & 1);
    // Gather the message's 512-float pieces out of the tile-major ring.
    const float *par = h->ring + (size_t)last * ring_parity_floats(h);
    const int64_t full = h->d / kRingTile, rem = h->d % kRingTile;
    hipError_t st = hipSuccess;
    if (full > 0)
        st = hipMemcpy2DAsync(dst_host, kRingTile * sizeof(float), par + (size_t)slot * kRingTile,
                              (size_t)h->e2 * kRingTile * sizeof(float), kRingTile * sizeof(float),
                              (size_t)full, hipMemcpyDeviceToHost, h->stream);
    if (st == hipSuccess && rem > 0)
        st = hipMemcpyAsync(dst_host + full * kRingTile,
                            par + ((size_t)full * h->e2 + slot) * kRingTile, rem * sizeof(float),
                            hipMemcpyDeviceToHost, h->stream);
    if (st == hipSuccess) st = hipStreamSynchronize(h->stream);
    return st == hipSuccess ? RELAYSUM_OK : hip_fail(h, st, "get_message");
}

}  // extern "C"
