// Host-side tree structures of the RelaySum library: the check that an edge
// list is a tree, its CSR form, and the plan that cuts a tree into clusters
// for the cluster kernels.  Plain C++ (no HIP), so that CPU tests can build
// it on its own, with sanitizers.
#pragma once

#include <algorithm>
#include <cstdint>
#include <utility>
#include <vector>

#include "relaysum.h"

// CSR form of a tree: slots row_ptr[i] .. row_ptr[i+1]-1 are the directed
// edges i -> col[s], col ascending; rev[s] is the slot of the reverse edge
// and src[s] = i.  e2 = 2(n-1) directed edges.
struct Csr {
    int32_t e2 = 0;
    std::vector<int32_t> row_ptr, col, rev, src;
};

// Checks that the edges form a tree on n workers and builds its CSR form.
inline int build_csr(int32_t n, const int32_t *edges, int32_t num_edges, Csr &tr) {
    if (num_edges > 0 && !edges) return RELAYSUM_ERR_INVALID_ARG;
    if (num_edges != n - 1) return RELAYSUM_ERR_NOT_A_TREE;
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
    tr.e2 = (int32_t)dir.size();
    tr.row_ptr.assign(n + 1, 0);
    tr.col.resize(tr.e2);
    tr.src.resize(tr.e2);
    tr.rev.resize(tr.e2);
    for (int32_t s = 0; s < tr.e2; ++s) {
        tr.src[s] = dir[s].first;
        tr.col[s] = dir[s].second;
        tr.row_ptr[dir[s].first + 1]++;
    }
    for (int32_t i = 0; i < n; ++i) tr.row_ptr[i + 1] += tr.row_ptr[i];
    for (int32_t s = 0; s < tr.e2; ++s) {
        const int32_t j = tr.col[s], i = tr.src[s];
        const auto b = tr.col.begin() + tr.row_ptr[j], e = tr.col.begin() + tr.row_ptr[j + 1];
        tr.rev[s] = (int32_t)(std::lower_bound(b, e, i) - tr.col.begin());
    }
    return RELAYSUM_OK;
}

// Cluster plan of a single tree: clusters of at most `cap` workers made of
// connected subtrees.  With worker 0 as the root, each worker, children
// before parents, keeps the open subtrees of its children that still fit,
// smallest first, and cuts the edges to the others.  The ends of the edges
// between clusters are the boundary workers.
// Workers of more than `hub_deg` neighbours (hubs) join no cluster: the
// clusters are planned on the forest the other workers form, and a hub's
// payload and out-messages come from a kernel of their own before the
// cluster kernel, so that a member reads a hub's message from the ring in
// its place in the sum.  A hub is a boundary worker whose sum the
// completion takes from the start.
//   members  [count][cap] worker ids of each cluster, -1 past its size
//   lslot    [e2] LDS slot of a message inside its cluster (0 .. slots-1,
//            distinct within a cluster), -2 for a message from a hub to a
//            member (read from the ring), -1 for any other message
//   bidx     [n] index of a boundary worker in bnd, -1 otherwise
//   bnd      the boundary workers (hubs included), ascending
//   rpos     [e2] ring position of each slot, a permutation of 0 .. e2-1
//            that puts each cluster's out-messages side by side, the hubs'
//            after all clusters'
//   bfirst   [nb] for each boundary worker, the index in its neighbour list
//            of its first neighbour that is neither in its cluster nor a
//            hub (0 for a hub)
//   nhubs    the hubs
struct ClusterPlan {
    int32_t count = 0, slots = 0, nhubs = 0;
    std::vector<int32_t> members, lslot, bidx, bnd, rpos, bfirst;
};

inline void plan_clusters(int32_t n, const Csr &tr, int cap, ClusterPlan &pl,
                          int32_t hub_deg = INT32_MAX) {
    const auto hub = [&](int32_t v) { return tr.row_ptr[v + 1] - tr.row_ptr[v] > hub_deg; };
    std::vector<int32_t> parent(n, -1), order, open(n, 0), cid(n, -1);
    std::vector<char> seen(n, 0), cut(n, 0);
    order.reserve(n);
    std::vector<int32_t> stack{0};
    seen[0] = 1;
    while (!stack.empty()) {
        const int32_t v = stack.back();
        stack.pop_back();
        order.push_back(v);
        for (int32_t q = tr.row_ptr[v]; q < tr.row_ptr[v + 1]; ++q) {
            const int32_t w = tr.col[q];
            if (!seen[w]) {
                seen[w] = 1;
                parent[w] = v;
                stack.push_back(w);
            }
        }
    }
    std::vector<std::pair<int32_t, int32_t>> kids;
    for (auto it = order.rbegin(); it != order.rend(); ++it) {
        const int32_t v = *it;
        if (hub(v)) continue;   // no subtree: its children start their own
        kids.clear();
        for (int32_t q = tr.row_ptr[v]; q < tr.row_ptr[v + 1]; ++q)
            if (parent[tr.col[q]] == v && !hub(tr.col[q]))
                kids.emplace_back(open[tr.col[q]], tr.col[q]);
        std::sort(kids.begin(), kids.end());
        int32_t size = 1;
        for (const auto &kw : kids) {
            if (size + kw.first <= cap) size += kw.first;
            else cut[kw.second] = 1;
        }
        open[v] = size;
    }
    // The components left by the cuts (the preorder lists every worker after
    // its parent), then packed into clusters of at most `cap` workers,
    // largest first, each into the first cluster with room: a cluster may
    // hold several components, which fills more of its workgroup's waves and
    // can only turn cut edges into inner ones.
    int32_t ncomp = 0;
    for (const int32_t v : order) {
        if (hub(v)) continue;
        cid[v] = (parent[v] < 0 || cut[v] || hub(parent[v])) ? ncomp++ : cid[parent[v]];
    }
    std::vector<int32_t> csize(ncomp, 0), corder(ncomp), load, group(ncomp);
    for (int32_t v = 0; v < n; ++v)
        if (cid[v] >= 0) ++csize[cid[v]];
    for (int32_t c = 0; c < ncomp; ++c) corder[c] = c;
    std::stable_sort(corder.begin(), corder.end(),
                     [&](int32_t a, int32_t b) { return csize[a] > csize[b]; });
    for (const int32_t c : corder) {
        size_t g = 0;
        while (g < load.size() && load[g] + csize[c] > cap) ++g;
        if (g == load.size()) load.push_back(0);
        load[g] += csize[c];
        group[c] = (int32_t)g;
    }
    for (int32_t v = 0; v < n; ++v)
        if (cid[v] >= 0) cid[v] = group[cid[v]];
    const int32_t count = (int32_t)load.size();
    pl.count = count;
    pl.nhubs = 0;
    pl.members.assign((size_t)count * cap, -1);
    std::vector<int32_t> fill(count, 0), nslots(count, 0);
    for (int32_t v = 0; v < n; ++v)
        if (cid[v] >= 0) pl.members[(size_t)cid[v] * cap + fill[cid[v]]++] = v;
    pl.lslot.assign(tr.e2, -1);
    pl.bidx.assign(n, -1);
    pl.bnd.clear();
    pl.bfirst.clear();
    for (int32_t v = 0; v < n; ++v) {
        int32_t first = -1;
        if (cid[v] < 0) {
            first = 0;
            ++pl.nhubs;
        } else {
            for (int32_t q = tr.row_ptr[v]; q < tr.row_ptr[v + 1]; ++q) {
                const int32_t w = tr.col[q];
                if (cid[w] == cid[v]) pl.lslot[q] = nslots[cid[v]]++;
                else if (cid[w] < 0) pl.lslot[tr.rev[q]] = -2;
                else if (first < 0) first = q - tr.row_ptr[v];
            }
        }
        if (first >= 0) {
            pl.bidx[v] = (int32_t)pl.bnd.size();
            pl.bnd.push_back(v);
            pl.bfirst.push_back(first);
        }
    }
    pl.slots = count ? *std::max_element(nslots.begin(), nslots.end()) : 0;
    // Ring positions: the messages out of each cluster's members side by
    // side, so that a workgroup's message pieces share a stretch of its ring
    // tile.
    pl.rpos.assign(tr.e2, -1);
    int32_t next = 0;
    for (int32_t c = 0; c < count; ++c)
        for (int32_t e = 0; e < cap; ++e) {
            const int32_t v = pl.members[(size_t)c * cap + e];
            if (v < 0) break;
            for (int32_t q = tr.row_ptr[v]; q < tr.row_ptr[v + 1]; ++q) pl.rpos[q] = next++;
        }
    for (int32_t v = 0; v < n; ++v)
        if (cid[v] < 0)
            for (int32_t q = tr.row_ptr[v]; q < tr.row_ptr[v + 1]; ++q) pl.rpos[q] = next++;
}

// Cluster plan of double binary trees: one set of clusters for both trees
// (a worker's row holds both trees' coordinates, so one workgroup reads it
// once for both).  The clusters are the cheapest of three candidates: tree
// A's cluster plan, tree B's, and runs of `cap` consecutive worker ids (the
// paper's pairs of trees are built on ranks, where such runs cut few edges
// of either tree).  The cost counts, per boundary worker (one with a
// neighbour in another cluster in either tree), the rows a completion
// launch moves: its partial sums written and read (one row) and, per tree,
// the messages from its first neighbour in another cluster on (half a row
// each: a tree's message carries half the coordinates).
//   members  [count][cap] worker ids of each cluster, -1 past its size
//   lslot[k] [e2 of tree k] LDS slot of a message of tree k inside its
//            cluster (distinct within the cluster and tree), -1 across
//   rpos[k]  [e2 of tree k] ring position of a slot of tree k, a permutation
//            putting each cluster's out-messages side by side
//   bidx     [n] index of a boundary worker in bnd, -1 otherwise
//   bnd      the boundary workers, ascending
//   bfirst[k][nb] index in tree k's neighbour list of the first neighbour
//            in another cluster, or the degree when there is none
struct DualPlan {
    int32_t count = 0, slots[2] = {0, 0};
    std::vector<int32_t> members, bidx, bnd;
    std::vector<int32_t> lslot[2], rpos[2], bfirst[2];
};

inline void plan_clusters_dual(int32_t n, const Csr &ta, const Csr &tb, int cap, DualPlan &pl) {
    const Csr *tr[2] = {&ta, &tb};
    // Candidate cluster ids.
    std::vector<std::vector<int32_t>> cands;
    for (const Csr *t : tr) {
        ClusterPlan p;
        plan_clusters(n, *t, cap, p);
        std::vector<int32_t> cid(n, -1);
        for (int32_t c = 0; c < p.count; ++c)
            for (int32_t e = 0; e < cap; ++e) {
                const int32_t v = p.members[(size_t)c * cap + e];
                if (v >= 0) cid[v] = c;
            }
        cands.push_back(std::move(cid));
    }
    {
        std::vector<int32_t> cid(n);
        for (int32_t v = 0; v < n; ++v) cid[v] = v / cap;
        cands.push_back(std::move(cid));
    }
    auto first_cross = [&](const Csr &t, const std::vector<int32_t> &cid, int32_t v) {
        for (int32_t q = t.row_ptr[v]; q < t.row_ptr[v + 1]; ++q)
            if (cid[t.col[q]] != cid[v]) return q - t.row_ptr[v];
        return t.row_ptr[v + 1] - t.row_ptr[v];
    };
    int64_t best_cost = -1;
    int32_t best_count = 0;
    size_t best = 0;
    for (size_t c = 0; c < cands.size(); ++c) {
        int64_t cost = 0;   // in half rows (a message of one tree)
        for (int32_t v = 0; v < n; ++v) {
            int64_t r = 0;
            bool boundary = false;
            for (const Csr *t : tr) {
                const int32_t deg = t->row_ptr[v + 1] - t->row_ptr[v];
                const int32_t f = first_cross(*t, cands[c], v);
                if (f < deg) boundary = true;
                r += deg - f;
            }
            if (boundary) cost += 4 + r;   // partial sums written and read: two rows
        }
        const int32_t count = *std::max_element(cands[c].begin(), cands[c].end()) + 1;
        if (best_cost < 0 || cost < best_cost || (cost == best_cost && count < best_count)) {
            best_cost = cost;
            best_count = count;
            best = c;
        }
    }
    const std::vector<int32_t> &cid = cands[best];
    pl.count = best_count;
    pl.members.assign((size_t)pl.count * cap, -1);
    std::vector<int32_t> fill(pl.count, 0);
    for (int32_t v = 0; v < n; ++v) pl.members[(size_t)cid[v] * cap + fill[cid[v]]++] = v;
    for (int k = 0; k < 2; ++k) {
        const Csr &t = *tr[k];
        std::vector<int32_t> nslots(pl.count, 0);
        pl.lslot[k].assign(t.e2, -1);
        for (int32_t v = 0; v < n; ++v)
            for (int32_t q = t.row_ptr[v]; q < t.row_ptr[v + 1]; ++q)
                if (cid[t.col[q]] == cid[v]) pl.lslot[k][q] = nslots[cid[v]]++;
        pl.slots[k] = pl.count ? *std::max_element(nslots.begin(), nslots.end()) : 0;
        pl.rpos[k].assign(t.e2, -1);
        int32_t next = 0;
        for (int32_t c = 0; c < pl.count; ++c)
            for (int32_t e = 0; e < cap; ++e) {
                const int32_t v = pl.members[(size_t)c * cap + e];
                if (v < 0) break;
                for (int32_t q = t.row_ptr[v]; q < t.row_ptr[v + 1]; ++q) pl.rpos[k][q] = next++;
            }
        pl.bfirst[k].clear();
    }
    pl.bidx.assign(n, -1);
    pl.bnd.clear();
    for (int32_t v = 0; v < n; ++v) {
        const int32_t fa = first_cross(ta, cid, v), fb = first_cross(tb, cid, v);
        if (fa < ta.row_ptr[v + 1] - ta.row_ptr[v] || fb < tb.row_ptr[v + 1] - tb.row_ptr[v]) {
            pl.bidx[v] = (int32_t)pl.bnd.size();
            pl.bnd.push_back(v);
            pl.bfirst[0].push_back(fa);
            pl.bfirst[1].push_back(fb);
        }
    }
}
