// CPU check of the library's host-side tree code (tree_plan.hpp): the tree
// validation and CSR form, and the cluster plan of the cluster kernels.
// Built with AddressSanitizer and UndefinedBehaviorSanitizer by
// tests/test_sanitize.py.  Prints "ok <trees checked>" and exits 0, or names
// the first broken invariant and exits 1.
#include <cstdio>
#include <cstdlib>
#include <set>
#include <vector>

#include "../../paper_2110_04175_amd/csrc/tree_plan.hpp"

namespace {

int failures = 0;
long checked = 0;

#define CHECK(cond, ...)                                              \
    do {                                                              \
        if (!(cond)) {                                                \
            std::fprintf(stderr, "FAIL %s:%d: %s: ", __FILE__, __LINE__, #cond); \
            std::fprintf(stderr, __VA_ARGS__);                        \
            std::fprintf(stderr, "\n");                               \
            ++failures;                                               \
            return;                                                   \
        }                                                             \
    } while (0)

uint64_t rng_state = 0x9e3779b97f4a7c15ull;
uint64_t next_u64() {   // xorshift64*
    rng_state ^= rng_state >> 12;
    rng_state ^= rng_state << 25;
    rng_state ^= rng_state >> 27;
    return rng_state * 2685821657736338717ull;
}

// Tree of a Pruefer sequence (smallest-leaf decoding), as an edge list.
std::vector<int32_t> pruefer_tree(int n, const std::vector<int> &seq) {
    std::vector<int32_t> e;
    if (n == 1) return e;
    std::vector<int> deg(n, 1);
    for (int v : seq) ++deg[v];
    std::set<int> leaves;
    for (int v = 0; v < n; ++v)
        if (deg[v] == 1) leaves.insert(v);
    for (int v : seq) {
        const int l = *leaves.begin();
        leaves.erase(leaves.begin());
        e.push_back(l);
        e.push_back(v);
        if (--deg[v] == 1) leaves.insert(v);
    }
    const int a = *leaves.begin(), b = *leaves.rbegin();
    e.push_back(a);
    e.push_back(b);
    return e;
}

void check_csr(int n, const std::vector<int32_t> &edges, const Csr &t) {
    const int e2 = 2 * (n - 1);
    CHECK(t.e2 == e2, "e2 %d", t.e2);
    CHECK((int)t.row_ptr.size() == n + 1 && t.row_ptr[0] == 0 && t.row_ptr[n] == e2, "row_ptr ends");
    CHECK((int)t.col.size() == e2 && (int)t.rev.size() == e2 && (int)t.src.size() == e2, "sizes");
    for (int i = 0; i < n; ++i) {
        CHECK(t.row_ptr[i] <= t.row_ptr[i + 1], "row_ptr not monotone at %d", i);
        for (int s = t.row_ptr[i]; s < t.row_ptr[i + 1]; ++s) {
            CHECK(t.src[s] == i, "src[%d]", s);
            CHECK(t.col[s] >= 0 && t.col[s] < n && t.col[s] != i, "col[%d]", s);
            if (s > t.row_ptr[i]) CHECK(t.col[s - 1] < t.col[s], "neighbours of %d not ascending", i);
            CHECK(t.rev[s] >= 0 && t.rev[s] < e2, "rev[%d] out of range", s);
            CHECK(t.rev[t.rev[s]] == s, "rev is not an involution at %d", s);
            CHECK(t.src[t.rev[s]] == t.col[s] && t.col[t.rev[s]] == i, "rev[%d] is not the reverse edge", s);
        }
    }
    std::set<std::pair<int, int>> want, got;
    for (size_t k = 0; k < edges.size(); k += 2)
        want.insert({std::min(edges[k], edges[k + 1]), std::max(edges[k], edges[k + 1])});
    for (int s = 0; s < e2; ++s)
        if (t.src[s] < t.col[s]) got.insert({t.src[s], t.col[s]});
    CHECK(want == got, "the CSR form holds other edges than the input");
}

// hub_deg: workers of more neighbours are hubs, in no cluster, boundary
// workers whose completion starts at their first neighbour; a member reads a
// hub's message from the ring (lslot -2) and counts no hub as a cut.
void check_plan(int n, const Csr &t, int cap, int32_t hub_deg, const ClusterPlan &pl) {
    CHECK(pl.count >= 1 && (int)pl.members.size() == pl.count * cap, "members size");
    std::vector<char> hub(n, 0);
    int nhubs = 0;
    for (int v = 0; v < n; ++v) {
        hub[v] = t.row_ptr[v + 1] - t.row_ptr[v] > hub_deg;
        nhubs += hub[v];
    }
    CHECK(pl.nhubs == nhubs, "nhubs %d, want %d", pl.nhubs, nhubs);
    std::vector<int> cid(n, -1);
    for (int c = 0; c < pl.count; ++c) {
        int size = 0;
        bool ended = false;
        for (int e = 0; e < cap; ++e) {
            const int v = pl.members[(size_t)c * cap + e];
            if (v < 0) { ended = true; continue; }
            CHECK(!ended, "cluster %d: a member after the padding", c);
            CHECK(v < n, "cluster %d: member %d out of range", c, v);
            CHECK(!hub[v], "hub %d in cluster %d", v, c);
            CHECK(cid[v] < 0, "worker %d in two clusters", v);
            cid[v] = c;
            ++size;
        }
        CHECK(size >= 1 && size <= cap, "cluster %d has %d members", c, size);
    }
    for (int v = 0; v < n; ++v) CHECK(hub[v] || cid[v] >= 0, "worker %d in no cluster", v);
    CHECK((int)pl.lslot.size() == t.e2 && (int)pl.rpos.size() == t.e2, "slot table sizes");
    std::vector<std::set<int>> inner(pl.count);
    std::vector<int> inner_count(pl.count, 0);
    for (int s = 0; s < t.e2; ++s) {
        const int u = t.src[s], w = t.col[s];
        const bool same = !hub[u] && !hub[w] && cid[u] == cid[w];
        if (hub[u] && !hub[w]) {
            CHECK(pl.lslot[s] == -2, "lslot[%d] = %d for a message from a hub", s, pl.lslot[s]);
            continue;
        }
        CHECK(same == (pl.lslot[s] >= 0) && (same || pl.lslot[s] == -1), "lslot[%d] = %d for %s message",
              s, pl.lslot[s], same ? "an inner" : "a cut");
        if (same) {
            inner[cid[u]].insert(pl.lslot[s]);
            ++inner_count[cid[u]];
        }
    }
    int slots = 0;
    for (int c = 0; c < pl.count; ++c) {
        CHECK((int)inner[c].size() == inner_count[c], "cluster %d: two messages share an LDS slot", c);
        if (inner_count[c] > 0)
            CHECK(*inner[c].begin() == 0 && *inner[c].rbegin() == inner_count[c] - 1,
                  "cluster %d: LDS slots are not 0 .. %d", c, inner_count[c] - 1);
        slots = std::max(slots, inner_count[c]);
    }
    CHECK(pl.slots == slots, "slots %d, largest cluster has %d", pl.slots, slots);
    // Boundary workers: the hubs (from their first neighbour) and the ends
    // of the cut edges between clusters, ascending, with the index of their
    // first neighbour in another cluster.
    std::vector<int> bnd;
    std::vector<int> first;
    for (int v = 0; v < n; ++v) {
        int f = hub[v] ? 0 : -1;
        if (!hub[v])
            for (int s = t.row_ptr[v]; s < t.row_ptr[v + 1]; ++s)
                if (!hub[t.col[s]] && cid[t.col[s]] != cid[v]) { f = s - t.row_ptr[v]; break; }
        if (f >= 0) { bnd.push_back(v); first.push_back(f); }
    }
    CHECK(pl.bnd == std::vector<int32_t>(bnd.begin(), bnd.end()), "boundary set");
    CHECK(pl.bfirst == std::vector<int32_t>(first.begin(), first.end()), "first cut neighbour");
    CHECK((int)pl.bidx.size() == n, "bidx size");
    for (int v = 0; v < n; ++v) {
        const int b = pl.bidx[v];
        if (b >= 0) CHECK(b < (int)bnd.size() && bnd[b] == v, "bidx[%d]", v);
        else CHECK(!std::binary_search(bnd.begin(), bnd.end(), v), "boundary worker %d without bidx", v);
    }
    // Ring positions: a permutation of the slots, the out-messages of each
    // cluster's members in one contiguous range, clusters in order, the
    // hubs' out-messages after them.
    std::vector<int> seen(t.e2, 0);
    for (int s = 0; s < t.e2; ++s) {
        CHECK(pl.rpos[s] >= 0 && pl.rpos[s] < t.e2 && !seen[pl.rpos[s]], "rpos is not a permutation at %d", s);
        seen[pl.rpos[s]] = 1;
    }
    int expect = 0;
    for (int c = 0; c < pl.count; ++c) {
        std::vector<int> pos;
        for (int e = 0; e < cap; ++e) {
            const int v = pl.members[(size_t)c * cap + e];
            if (v < 0) break;
            for (int s = t.row_ptr[v]; s < t.row_ptr[v + 1]; ++s) pos.push_back(pl.rpos[s]);
        }
        std::sort(pos.begin(), pos.end());
        for (size_t k = 0; k < pos.size(); ++k)
            CHECK(pos[k] == expect + (int)k, "cluster %d: ring positions not contiguous", c);
        expect += (int)pos.size();
    }
    for (int v = 0; v < n; ++v)
        if (hub[v])
            for (int s = t.row_ptr[v]; s < t.row_ptr[v + 1]; ++s)
                CHECK(pl.rpos[s] >= expect, "hub %d: ring position inside the clusters' range", v);
}

// The two-tree plan: every worker in exactly one cluster; per tree, LDS
// slots bijective within each cluster and ring positions a permutation with
// each cluster's out-messages together; the boundary set the workers with a
// cut edge in either tree, with each tree's first cut neighbour (or the
// degree when the tree has none).
void check_dual(int n, const Csr &ta, const Csr &tb, int cap, const DualPlan &pl) {
    CHECK(pl.count >= 1 && (int)pl.members.size() == pl.count * cap, "dual members size");
    std::vector<int> cid(n, -1);
    for (int c = 0; c < pl.count; ++c)
        for (int e = 0; e < cap; ++e) {
            const int v = pl.members[(size_t)c * cap + e];
            if (v < 0) continue;
            CHECK(v < n && cid[v] < 0, "dual: worker %d placed twice or out of range", v);
            cid[v] = c;
        }
    for (int v = 0; v < n; ++v) CHECK(cid[v] >= 0, "dual: worker %d in no cluster", v);
    const Csr *tr[2] = {&ta, &tb};
    for (int k = 0; k < 2; ++k) {
        const Csr &t = *tr[k];
        std::vector<std::set<int>> inner(pl.count);
        std::vector<int> cnt(pl.count, 0);
        for (int s = 0; s < t.e2; ++s) {
            const bool same = cid[t.src[s]] == cid[t.col[s]];
            CHECK(same == (pl.lslot[k][s] >= 0), "dual tree %d: lslot[%d]", k, s);
            if (same) { inner[cid[t.src[s]]].insert(pl.lslot[k][s]); ++cnt[cid[t.src[s]]]; }
        }
        int slots = 0;
        for (int c = 0; c < pl.count; ++c) {
            CHECK((int)inner[c].size() == cnt[c], "dual tree %d cluster %d: shared LDS slot", k, c);
            if (cnt[c]) CHECK(*inner[c].rbegin() == cnt[c] - 1, "dual tree %d cluster %d: slots not dense", k, c);
            slots = std::max(slots, cnt[c]);
        }
        CHECK(pl.slots[k] == slots, "dual tree %d: slots", k);
        std::vector<int> seen(t.e2, 0);
        for (int s = 0; s < t.e2; ++s) {
            CHECK(pl.rpos[k][s] >= 0 && pl.rpos[k][s] < t.e2 && !seen[pl.rpos[k][s]], "dual tree %d: rpos", k);
            seen[pl.rpos[k][s]] = 1;
        }
    }
    std::vector<int32_t> bnd, fa, fb;
    for (int v = 0; v < n; ++v) {
        int f[2];
        for (int k = 0; k < 2; ++k) {
            const Csr &t = *tr[k];
            f[k] = t.row_ptr[v + 1] - t.row_ptr[v];
            for (int s = t.row_ptr[v]; s < t.row_ptr[v + 1]; ++s)
                if (cid[t.col[s]] != cid[v]) { f[k] = s - t.row_ptr[v]; break; }
        }
        if (f[0] < ta.row_ptr[v + 1] - ta.row_ptr[v] || f[1] < tb.row_ptr[v + 1] - tb.row_ptr[v]) {
            bnd.push_back(v); fa.push_back(f[0]); fb.push_back(f[1]);
        }
    }
    CHECK(pl.bnd == bnd && pl.bfirst[0] == fa && pl.bfirst[1] == fb, "dual boundary set");
    for (int v = 0; v < n; ++v) {
        const int b = pl.bidx[v];
        if (b >= 0) CHECK(b < (int)bnd.size() && bnd[b] == v, "dual bidx[%d]", v);
    }
}

void check_pair(int n, const std::vector<int32_t> &ea, const std::vector<int32_t> &eb, int cap) {
    Csr ta, tb;
    if (build_csr(n, ea.empty() ? nullptr : ea.data(), (int32_t)ea.size() / 2, ta) != RELAYSUM_OK ||
        build_csr(n, eb.empty() ? nullptr : eb.data(), (int32_t)eb.size() / 2, tb) != RELAYSUM_OK) {
        std::fprintf(stderr, "FAIL: a pair of trees of %d workers rejected\n", n);
        ++failures;
        return;
    }
    DualPlan pl;
    plan_clusters_dual(n, ta, tb, cap, pl);
    check_dual(n, ta, tb, cap, pl);
    ++checked;
}

void check_tree(int n, const std::vector<int32_t> &edges, std::initializer_list<int> caps) {
    Csr t;
    const int rc = build_csr(n, edges.empty() ? nullptr : edges.data(), (int32_t)edges.size() / 2, t);
    if (rc != RELAYSUM_OK) {
        std::fprintf(stderr, "FAIL: a tree of %d workers rejected (%d)\n", n, rc);
        ++failures;
        return;
    }
    check_csr(n, edges, t);
    for (int cap : caps) {
        ClusterPlan pl;
        plan_clusters(n, t, cap, pl);
        check_plan(n, t, cap, INT32_MAX, pl);
        // Hubs: workers of more than 1 (every inner worker), 2 or 8 neighbours.
        for (int32_t hub_deg : {1, 2, 8}) {
            ClusterPlan ph;
            plan_clusters(n, t, cap, ph, hub_deg);
            check_plan(n, t, cap, hub_deg, ph);
        }
    }
    ++checked;
}

void check_rejected(int n, const std::vector<int32_t> &edges, int num_edges, int want) {
    Csr t;
    const int rc = build_csr(n, edges.empty() ? nullptr : edges.data(), num_edges, t);
    if (rc != want) {
        std::fprintf(stderr, "FAIL: bad edge list of %d workers gave %d, want %d\n", n, rc, want);
        ++failures;
    }
}

}  // namespace

int main() {
    // Every labelled tree of up to 7 workers (n^(n-2) Pruefer sequences),
    // planned into clusters of 1 to 4 and 16 workers.
    for (int n = 1; n <= 7; ++n) {
        const int len = n >= 2 ? n - 2 : 0;
        long total = 1;
        for (int k = 0; k < len; ++k) total *= n;
        for (long code = 0; code < total; ++code) {
            std::vector<int> seq(len);
            long c = code;
            for (int k = 0; k < len; ++k) { seq[k] = (int)(c % n); c /= n; }
            check_tree(n, pruefer_tree(n, seq), {1, 2, 3, 4, 16});
        }
    }
    // Random trees up to 4096 workers, and chains, stars, brooms and heaps.
    for (int k = 0; k < 300; ++k) {
        const int n = 2 + (int)(next_u64() % 4095);
        std::vector<int> seq(n - 2);
        for (int &v : seq) v = (int)(next_u64() % n);
        check_tree(n, pruefer_tree(n, seq), {16});
    }
    for (int n : {2, 3, 17, 33, 64, 100, 256, 300, 1000, 4096, 5000}) {
        std::vector<int32_t> chain, star, heap, broom;
        for (int i = 1; i < n; ++i) {
            chain.insert(chain.end(), {i - 1, i});
            star.insert(star.end(), {0, i});
            heap.insert(heap.end(), {(i - 1) / 2, i});
            broom.insert(broom.end(), {i < n - 12 ? i - 1 : n - 13 < 0 ? 0 : n - 13, i});
        }
        check_tree(n, chain, {16});
        check_tree(n, star, {16});
        check_tree(n, heap, {16});
        if (n > 13) check_tree(n, broom, {16});
    }
    // Pairs of trees for the double-tree plan: random pairs, chain and star,
    // and in-order binary trees with their rank-shifted copies.
    for (int k = 0; k < 200; ++k) {
        const int n = 2 + (int)(next_u64() % 600);
        std::vector<int> sa(n - 2), sb(n - 2);
        for (int &v : sa) v = (int)(next_u64() % n);
        for (int &v : sb) v = (int)(next_u64() % n);
        check_pair(n, pruefer_tree(n, sa), pruefer_tree(n, sb), k % 2 ? 16 : 5);
    }
    for (int n : {65, 100, 128, 200, 1000}) {
        std::vector<int32_t> chain, star, ina, inb;
        for (int i = 1; i < n; ++i) {
            chain.insert(chain.end(), {i - 1, i});
            star.insert(star.end(), {0, i});
        }
        check_pair(n, star, chain, 16);
        check_pair(n, chain, chain, 16);
        // In-order binary tree on ranks 0..n-1 (parent of a range's middle
        // is the middle of the enclosing range) and its copy shifted by one.
        std::vector<std::pair<int, int>> todo{{0, n - 1}};
        std::vector<int> par_of_range{-1};
        for (size_t q = 0; q < todo.size(); ++q) {
            const int lo = todo[q].first, hi = todo[q].second, p = par_of_range[q];
            if (lo > hi) continue;
            const int mid = (lo + hi) / 2;
            if (p >= 0) { ina.insert(ina.end(), {p, mid}); inb.insert(inb.end(), {(p + 1) % n, (mid + 1) % n}); }
            todo.push_back({lo, mid - 1}); par_of_range.push_back(mid);
            todo.push_back({mid + 1, hi}); par_of_range.push_back(mid);
        }
        check_pair(n, ina, inb, 16);
    }
    // Edge lists that are not trees.
    check_rejected(3, {0, 1, 1, 1}, 2, RELAYSUM_ERR_NOT_A_TREE);       // self loop
    check_rejected(3, {0, 1, 0, 1}, 2, RELAYSUM_ERR_NOT_A_TREE);       // duplicate
    check_rejected(3, {1, 0, 0, 1}, 2, RELAYSUM_ERR_NOT_A_TREE);       // duplicate, reversed
    check_rejected(4, {0, 1, 1, 2, 2, 0}, 3, RELAYSUM_ERR_NOT_A_TREE); // cycle
    check_rejected(3, {0, 1, 1, 3}, 2, RELAYSUM_ERR_NOT_A_TREE);       // id out of range
    check_rejected(3, {0, -1, 1, 2}, 2, RELAYSUM_ERR_NOT_A_TREE);      // negative id
    check_rejected(3, {0, 1}, 1, RELAYSUM_ERR_NOT_A_TREE);             // too few edges
    check_rejected(3, {}, 2, RELAYSUM_ERR_INVALID_ARG);                // NULL edges
    if (failures) {
        std::fprintf(stderr, "%d failures\n", failures);
        return 1;
    }
    std::printf("ok %ld trees\n", checked);
    return 0;
}
