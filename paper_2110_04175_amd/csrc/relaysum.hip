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
//   ring                float[2][2E][ring_stride]: slot t&1 receives the
//                       messages of round t while slot (t-1)&1 holds those
//                       of round t-1; ring_stride = d rounded up to 64 floats
//                       so every message row starts on a 256-byte boundary
//   counts              int32[2][2E] double-buffered like the ring, nbar[n]
//   tree                CSR: row_ptr[n+1]; slots row_ptr[i]..row_ptr[i+1]-1
//                       are the directed edges i->col[s], col ascending;
//                       rev[s] is the slot of the reverse edge; src[s] = i
//
// Tile kernel (trees up to a few hundred workers).  A workgroup owns a tile
// of 64*V consecutive coordinates of every row; each wave owns whole workers
// (worker i belongs to wave i mod W).  Phase 1: a wave streams x_i, g_i,
// mom_i and the previous messages into i, forms the half-step xh_i (kept in
// registers), writes mom_i and the messages i->j to HBM and to an LDS tile
// [2E][64*V].  After a barrier, phase 2 forms each average from xh_i and the
// LDS copies of the new messages into i and writes x_i.  New messages are
// therefore read back from LDS, never from HBM, and every HBM byte of the
// round is touched exactly once.
//
// Two-pass path (larger trees, whose message tile does not fit in LDS): one
// small launch relays the counters, one writes xh into x together with the
// new messages, one forms the averages from x and the new messages.
//
// Arithmetic: one IEEE binary32 rounding per operation, contraction off, sums
// start from xh_i and add neighbours in ascending id, the average is a
// correctly rounded division.  Results do not depend on V, the tile or grid.

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
constexpr int kMaxDegInRegs = 4;    // previous messages into a worker kept in VGPRs
constexpr int64_t kRowAlign = 64;   // message rows padded to 64 floats (256 B)

template <int V>
struct vf {
    float v[V];
};

typedef float f4_t __attribute__((ext_vector_type(4)));

template <int V>
__device__ __forceinline__ vf<V> load_v(const float *__restrict__ p) {
    vf<V> r;
    if constexpr (V == 4) {
        f4_t t = *reinterpret_cast<const f4_t *>(p);
        r.v[0] = t.x; r.v[1] = t.y; r.v[2] = t.z; r.v[3] = t.w;
    } else {
#pragma unroll
        for (int k = 0; k < V; ++k) r.v[k] = p[k];
    }
    return r;
}

template <int V>
__device__ __forceinline__ void store_v(float *__restrict__ p, const vf<V> &a) {
    if constexpr (V == 4) {
        f4_t t = {a.v[0], a.v[1], a.v[2], a.v[3]};
        *reinterpret_cast<f4_t *>(p) = t;
    } else {
#pragma unroll
        for (int k = 0; k < V; ++k) p[k] = a.v[k];
    }
}

template <int V>
__device__ __forceinline__ vf<V> zero_v() {
    vf<V> r;
#pragma unroll
    for (int k = 0; k < V; ++k) r.v[k] = 0.0f;
    return r;
}

template <int V>
__device__ __forceinline__ vf<V> add_v(const vf<V> &a, const vf<V> &b) {
    vf<V> r;
#pragma unroll
    for (int k = 0; k < V; ++k) r.v[k] = a.v[k] + b.v[k];
    return r;
}

// Local half-step of worker i on V coordinates (Alg. 1 line 3; App. D.2).
// With momentum: b <- beta*b + g; xh = x - lr*(g + beta*b).
template <int V, bool MOM>
__device__ __forceinline__ vf<V> half_step(const vf<V> &x, const vf<V> &g, vf<V> &b,
                                           float lr, float beta) {
    vf<V> xh;
#pragma unroll
    for (int k = 0; k < V; ++k) {
        if constexpr (MOM) {
            const float p = beta * b.v[k];
            const float bn = p + g.v[k];
            b.v[k] = bn;
            const float q = beta * bn;
            const float u = g.v[k] + q;
            const float s = lr * u;
            xh.v[k] = x.v[k] - s;
        } else {
            const float s = lr * g.v[k];
            xh.v[k] = x.v[k] - s;
        }
    }
    return xh;
}

struct RoundArgs {
    float *x;
    const float *g;
    float *mom;
    const float *ring_prev;   // messages of round t-1, [2E][ring_stride]
    float *ring_next;         // messages of round t
    int64_t ring_stride;      // floats between message rows
    int64_t d;                // floats per model row
    int64_t nchunks;          // d / V
    int64_t ntiles;           // ceil(nchunks / 64)
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

// Tile index handled by workgroup `b` on its k-th turn, or -1 when done.
// Workgroups are dispatched to the 8 XCDs round-robin (b mod 8), so the
// tiles are cut into 8 contiguous ranges, one per XCD: neighbouring tiles
// then run at the same time in the same L2, which holds the cache lines a
// tile boundary splits.
__device__ __forceinline__ int64_t tile_of(int64_t b, int64_t k, int64_t G, int64_t T) {
    if (G >= 8 && (G & 7) == 0) {
        const int64_t Q = G >> 3, xcd = b & 7, q = b >> 3;
        const int64_t per = (T + 7) >> 3;
        const int64_t t = xcd * per + q + k * Q;
        return (q + k * Q < per && t < T) ? t : -1;
    }
    const int64_t t = b + k * G;
    return t < T ? t : -1;
}

template <int V, int PW, bool MOM>
__global__ void __launch_bounds__(1024) relaysum_tile_kernel(RoundArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    int32_t *s_cnt = reinterpret_cast<int32_t *>(smem);
    int32_t *s_nbar = s_cnt + a.e2;
    const int hdr = ((a.e2 + a.n) * 4 + 15) & ~15;
    float *s_msg = reinterpret_cast<float *>(smem + hdr);   // [2E][64*V]

    relay_counts(a, s_cnt, s_nbar);
    if (blockIdx.x == 0) {
        for (int s = threadIdx.x; s < a.e2; s += blockDim.x) a.cnt_next[s] = s_cnt[s];
        for (int i = threadIdx.x; i < a.n; i += blockDim.x) a.nbar_out[i] = s_nbar[i];
    }

    const int lane = threadIdx.x & (kWave - 1);
    const int wave = uniform(threadIdx.x >> 6);
    const int W = blockDim.x >> 6;
    const int64_t G = gridDim.x;

    for (int64_t k = 0;; ++k) {
        const int64_t tile = tile_of(blockIdx.x, k, G, a.ntiles);
        if (tile < 0) break;
        const int64_t chunk = tile * kWave + lane;
        const bool ok = chunk < a.nchunks;
        const int64_t off = chunk * V;

        vf<V> xh[PW];
        // Phase 1: half-steps, momentum, outgoing messages.
#pragma unroll
        for (int p = 0; p < PW; ++p) {
            const int i = wave + p * W;
            if (i >= a.n) break;
            const int64_t row = (int64_t)i * a.d + off;
            vf<V> xv = zero_v<V>(), gv = zero_v<V>(), bv = zero_v<V>();
            if (ok) {
                xv = load_v<V>(a.x + row);
                gv = load_v<V>(a.g + row);
                if constexpr (MOM) bv = load_v<V>(a.mom + row);
            }
            const int s0 = uniform(a.row_ptr[i]);
            const int deg = uniform(a.row_ptr[i + 1]) - s0;
            vf<V> o[kMaxDegInRegs];
            if (deg <= kMaxDegInRegs) {
#pragma unroll
                for (int b = 0; b < kMaxDegInRegs; ++b) {
                    if (b < deg) {
                        const int in_slot = uniform(a.rev[s0 + b]);
                        o[b] = ok ? load_v<V>(a.ring_prev + in_slot * a.ring_stride + off)
                                  : zero_v<V>();
                    }
                }
            }
            xh[p] = half_step<V, MOM>(xv, gv, bv, a.lr, a.beta);
            if constexpr (MOM) {
                if (ok) store_v<V>(a.mom + row, bv);
            }
            if (deg <= kMaxDegInRegs) {
#pragma unroll
                for (int q = 0; q < kMaxDegInRegs; ++q) {
                    if (q < deg) {
                        vf<V> m = xh[p];
#pragma unroll
                        for (int b = 0; b < kMaxDegInRegs; ++b)
                            if (b < deg && b != q) m = add_v<V>(m, o[b]);
                        if (ok) store_v<V>(a.ring_next + (s0 + q) * a.ring_stride + off, m);
                        store_v<V>(s_msg + ((s0 + q) * kWave + lane) * V, m);
                    }
                }
            } else {
                for (int q = 0; q < deg; ++q) {
                    vf<V> m = xh[p];
                    for (int b = 0; b < deg; ++b) {
                        if (b == q) continue;
                        const int in_slot = uniform(a.rev[s0 + b]);
                        if (ok) m = add_v<V>(m, load_v<V>(a.ring_prev + in_slot * a.ring_stride + off));
                    }
                    if (ok) store_v<V>(a.ring_next + (s0 + q) * a.ring_stride + off, m);
                    store_v<V>(s_msg + ((s0 + q) * kWave + lane) * V, m);
                }
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
            vf<V> acc = xh[p];
            for (int q = 0; q < deg; ++q) {
                const int in_slot = uniform(a.rev[s0 + q]);
                acc = add_v<V>(acc, load_v<V>(s_msg + (in_slot * kWave + lane) * V));
            }
            const float nb = (float)s_nbar[i];
            vf<V> xn;
#pragma unroll
            for (int c = 0; c < V; ++c) xn.v[c] = acc.v[c] / nb;
            if (ok) store_v<V>(a.x + (int64_t)i * a.d + off, xn);
        }
        __syncthreads();
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

// Half-step and outgoing messages of worker blockIdx.y (grid-strided);
// the half-step is left in x for the averaging pass.
template <int V, bool MOM>
__global__ void __launch_bounds__(256) relaysum_pass_a(RoundArgs a) {
    for (int i = blockIdx.y; i < a.n; i += gridDim.y) {
        const int s0 = a.row_ptr[i];
        const int deg = a.row_ptr[i + 1] - s0;
        for (int64_t chunk = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; chunk < a.nchunks;
             chunk += (int64_t)gridDim.x * blockDim.x) {
            const int64_t off = chunk * V;
            const int64_t row = (int64_t)i * a.d + off;
            vf<V> xv = load_v<V>(a.x + row), gv = load_v<V>(a.g + row), bv = zero_v<V>();
            if constexpr (MOM) bv = load_v<V>(a.mom + row);
            const vf<V> xh = half_step<V, MOM>(xv, gv, bv, a.lr, a.beta);
            if constexpr (MOM) store_v<V>(a.mom + row, bv);
            for (int q = 0; q < deg; ++q) {
                vf<V> m = xh;
                for (int b = 0; b < deg; ++b) {
                    if (b == q) continue;
                    m = add_v<V>(m, load_v<V>(a.ring_prev + a.rev[s0 + b] * a.ring_stride + off));
                }
                store_v<V>(a.ring_next + (s0 + q) * a.ring_stride + off, m);
            }
            store_v<V>(a.x + row, xh);
        }
    }
}

template <int V>
__global__ void __launch_bounds__(256) relaysum_pass_b(RoundArgs a) {
    for (int i = blockIdx.y; i < a.n; i += gridDim.y) {
        const int s0 = a.row_ptr[i];
        const int deg = a.row_ptr[i + 1] - s0;
        const float nb = (float)a.nbar_out[i];
        for (int64_t chunk = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; chunk < a.nchunks;
             chunk += (int64_t)gridDim.x * blockDim.x) {
            const int64_t off = chunk * V;
            const int64_t row = (int64_t)i * a.d + off;
            vf<V> acc = load_v<V>(a.x + row);
            for (int q = 0; q < deg; ++q)
                acc = add_v<V>(acc, load_v<V>(a.ring_next + a.rev[s0 + q] * a.ring_stride + off));
            vf<V> xn;
#pragma unroll
            for (int c = 0; c < V; ++c) xn.v[c] = acc.v[c] / nb;
            store_v<V>(a.x + row, xn);
        }
    }
}

// ---- host side --------------------------------------------------------------

typedef void (*tile_fn)(RoundArgs);

// 128-bit lanes are used only while the [2E][256] message tile stays small
// (n <= 32, so at most two workers per wave); wider trees use 32-bit lanes.
template <bool MOM>
tile_fn pick_tile_v4(int pw) {
    switch (pw) {
        case 1: return relaysum_tile_kernel<4, 1, MOM>;
        case 2: return relaysum_tile_kernel<4, 2, MOM>;
        default: return nullptr;
    }
}

template <bool MOM>
tile_fn pick_tile_v1(int pw) {
    switch (pw) {
        case 1: return relaysum_tile_kernel<1, 1, MOM>;
        case 2: return relaysum_tile_kernel<1, 2, MOM>;
        case 4: return relaysum_tile_kernel<1, 4, MOM>;
        case 8: return relaysum_tile_kernel<1, 8, MOM>;
        case 16: return relaysum_tile_kernel<1, 16, MOM>;
        case 32: return relaysum_tile_kernel<1, 32, MOM>;
        default: return nullptr;
    }
}

constexpr size_t kLdsPreferV4 = 64 * 1024;      // keep >= 2 workgroups per CU

size_t tile_lds_bytes(int n, int e2, int V) {
    const size_t hdr = (((size_t)e2 + n) * 4 + 15) & ~(size_t)15;
    return hdr + (size_t)e2 * kWave * V * sizeof(float);
}

}  // namespace

struct relaysum_s {
    int32_t n = 0;
    int64_t d = 0;
    int32_t e2 = 0;
    std::vector<int32_t> row_ptr, col, rev, src;
    int32_t *d_topo = nullptr;   // row_ptr[n+1] | col[e2] | rev[e2] | src[e2]
    int32_t *d_counts = nullptr; // cnt[2][e2] | nbar[n]
    float *ring = nullptr;       // [2][e2][ring_stride]
    int64_t ring_stride = 0;
    int64_t t = 0;
    hipStream_t stream = nullptr;
    int device = 0;
    int cu_count = 256;
    int waves = 1;               // W: waves per workgroup of the tile kernel
    int pw = 1;                  // workers per wave (power of two)
    int tile_v = 0;              // 4 or 1 when the tile kernel fits, 0 = two-pass
    size_t lds_limit = 64 * 1024;
    struct Launch {
        tile_fn fn = nullptr;
        int64_t grid = 0;
        size_t lds = 0;
    } launch[2][2];              // [V == 4][momentum], filled on first use
    std::string err;
};

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

    // Tile plan: W waves per workgroup, pw workers per wave, V floats per lane.
    h->waves = std::min<int>(n, kMaxWaves);
    int pw = 1;
    while (pw * h->waves < n) pw *= 2;
    h->pw = pw;
    if (pw <= 32) {
        if (pw <= 2 && tile_lds_bytes(n, h->e2, 4) <= kLdsPreferV4) h->tile_v = 4;
        else if (tile_lds_bytes(n, h->e2, 1) <= h->lds_limit) h->tile_v = 1;
    }

    const size_t topo_ints = (size_t)(n + 1) + 3 * (size_t)h->e2;
    if (hipMalloc(&h->d_topo, topo_ints * sizeof(int32_t)) != hipSuccess ||
        hipMalloc(&h->d_counts, (2 * (size_t)h->e2 + n) * sizeof(int32_t)) != hipSuccess) {
        release(h);
        return RELAYSUM_ERR_OUT_OF_MEMORY;
    }
    h->ring_stride = (d + kRowAlign - 1) / kRowAlign * kRowAlign;
    if (h->e2 > 0 && d > 0) {
        const size_t bytes = 2 * (size_t)h->e2 * (size_t)h->ring_stride * sizeof(float);
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
                            2 * (size_t)h->e2 * (size_t)h->ring_stride * sizeof(float), h->stream);
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
    a.ring_stride = h->ring_stride;
    a.ring_prev = h->ring ? h->ring + (size_t)prev * h->e2 * h->ring_stride : nullptr;
    a.ring_next = h->ring ? h->ring + (size_t)next * h->e2 * h->ring_stride : nullptr;
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
        const int V = (h->tile_v == 4 && vec4) ? 4 : 1;
        a.nchunks = h->d / V;
        a.ntiles = (a.nchunks + kWave - 1) / kWave;
        const int threads = h->waves * kWave;
        relaysum_s::Launch &L = h->launch[V == 4][use_mom];
        if (!L.fn) {
            tile_fn fn = V == 4 ? (use_mom ? pick_tile_v4<true>(h->pw) : pick_tile_v4<false>(h->pw))
                                : (use_mom ? pick_tile_v1<true>(h->pw) : pick_tile_v1<false>(h->pw));
            if (!fn) return fail(h, RELAYSUM_ERR_INVALID_ARG, "no tile kernel for this tree");
            const size_t lds = tile_lds_bytes(h->n, h->e2, V);
            hipError_t st = hipFuncSetAttribute((const void *)fn,
                                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
            if (st != hipSuccess) return hip_fail(h, st, "hipFuncSetAttribute");
            int per_cu = 0;
            st = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, (const void *)fn, threads, lds);
            if (st != hipSuccess || per_cu < 1) {
                (void)hipGetLastError();
                per_cu = 1;
            }
            L.fn = fn;
            L.lds = lds;
            L.grid = (int64_t)per_cu * h->cu_count;
        }
        int64_t grid = std::min<int64_t>(L.grid, a.ntiles);
        if (grid >= 8) grid &= ~(int64_t)7;
        if (grid < 1) grid = 1;
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
    const float *row = h->ring + ((size_t)last * h->e2 + slot) * h->ring_stride;
    hipError_t st = hipMemcpyAsync(dst_host, row, (size_t)h->d * sizeof(float),
                                   hipMemcpyDeviceToHost, h->stream);
    if (st == hipSuccess) st = hipStreamSynchronize(h->stream);
    return st == hipSuccess ? RELAYSUM_OK : hip_fail(h, st, "get_message");
}

}  // extern "C"
