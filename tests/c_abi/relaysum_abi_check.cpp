// A consumer of librelaysum.so through include/relaysum.h alone: plain device
// pointers from the HIP runtime, no Python and no torch.  It runs the
// 3-worker chain worked by hand from Alg. 1 with the momentum of Appendix
// D.2 (values read from tests/golden/chain3_alg1_hand_worked.txt), checks the
// counters, messages and models of every round, the error codes of invalid
// calls, and that a double-tree handle equals two single-tree handles on the
// odd and even coordinates (Section 3), bit for bit.
//
//   relaysum_abi_check <path of chain3_alg1_hand_worked.txt>
//
// Prints one line per failed check and a summary; exit status 0 iff all pass.
#include <hip/hip_runtime_api.h>

#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <vector>

#include "relaysum.h"

static int g_checks = 0, g_failed = 0;

static void check(bool ok, const char *what) {
    ++g_checks;
    if (!ok) {
        ++g_failed;
        std::printf("FAILED: %s\n", what);
    }
}

static void hip_ok(hipError_t e, const char *what) {
    if (e != hipSuccess) {
        std::printf("HIP error in %s: %s\n", what, hipGetErrorString(e));
        std::exit(2);
    }
}

// "a/b" or "a" -> double.
static double frac(const std::string &tok) {
    const size_t p = tok.find('/');
    if (p == std::string::npos) return std::strtod(tok.c_str(), nullptr);
    return std::strtod(tok.substr(0, p).c_str(), nullptr) /
           std::strtod(tok.substr(p + 1).c_str(), nullptr);
}

static std::vector<double> values(const std::string &field) {
    std::vector<double> out;
    const size_t eq = field.find('=');
    std::string rest = field.substr(eq + 1);
    char *save = nullptr;
    std::vector<char> buf(rest.begin(), rest.end());
    buf.push_back('\0');
    for (char *t = strtok_r(buf.data(), " \t", &save); t; t = strtok_r(nullptr, " \t", &save))
        out.push_back(frac(t));
    return out;
}

struct Round { std::vector<double> m, c, nbar, x, mom; };
struct Case { std::vector<double> x0, g; double lr = 0, beta = 0; std::vector<Round> rounds; };

static bool read_case(const char *path, const char *name, Case &out) {
    FILE *f = std::fopen(path, "r");
    if (!f) return false;
    char line[1024];
    bool in = false;
    while (std::fgets(line, sizeof line, f)) {
        std::string s(line);
        while (!s.empty() && (s.back() == '\n' || s.back() == '\r')) s.pop_back();
        if (s.empty() || s[0] == '#') continue;
        if (s.rfind("case ", 0) == 0) { in = s.substr(5) == name; continue; }
        if (!in) continue;
        if (s.rfind("round ", 0) == 0) {
            Round r;
            size_t pos = s.find('|');
            while (pos != std::string::npos) {
                const size_t next = s.find('|', pos + 1);
                const std::string fld = s.substr(pos + 1, next == std::string::npos ? std::string::npos : next - pos - 1);
                const std::string key = fld.substr(fld.find_first_not_of(' '), fld.find('=') - fld.find_first_not_of(' '));
                const std::vector<double> v = values(fld);
                if (key.rfind("m ", 0) == 0) r.m = v;
                else if (key.rfind("c ", 0) == 0) r.c = v;
                else if (key.rfind("nbar", 0) == 0) r.nbar = v;
                else if (key.rfind("x ", 0) == 0) r.x = v;
                else if (key.rfind("mom", 0) == 0) r.mom = v;
                pos = next;
            }
            out.rounds.push_back(r);
        } else if (s.rfind("x0", 0) == 0) out.x0 = values(s);
        else if (s.rfind("g ", 0) == 0) out.g = values(s);
        else if (s.rfind("lr", 0) == 0) out.lr = values(s)[0];
        else if (s.rfind("beta", 0) == 0) out.beta = values(s)[0];
    }
    std::fclose(f);
    return !out.rounds.empty();
}

static bool close_to(double got, double want) {
    return std::fabs(got - want) <= 3e-7 * std::fmax(1.0, std::fabs(want));
}

static void hand_worked_chain(const char *fixture, const char *name) {
    Case c;
    check(read_case(fixture, name, c), "read the hand-worked fixture");
    if (c.rounds.empty()) return;
    const int32_t edges[4] = {0, 1, 1, 2};
    relaysum_t *h = nullptr;
    check(relaysum_create(3, 1, edges, 2, &h) == RELAYSUM_OK && h, "create the 3-worker chain");
    float *x, *g, *mom;
    hip_ok(hipMalloc((void **)&x, 3 * sizeof(float)), "hipMalloc");
    hip_ok(hipMalloc((void **)&g, 3 * sizeof(float)), "hipMalloc");
    hip_ok(hipMalloc((void **)&mom, 3 * sizeof(float)), "hipMalloc");
    float hx[3], hg[3], hm[3] = {0, 0, 0};
    for (int i = 0; i < 3; ++i) { hx[i] = (float)c.x0[i]; hg[i] = (float)c.g[i]; }
    hip_ok(hipMemcpy(x, hx, sizeof hx, hipMemcpyHostToDevice), "copy x0");
    hip_ok(hipMemcpy(g, hg, sizeof hg, hipMemcpyHostToDevice), "copy g");
    hip_ok(hipMemcpy(mom, hm, sizeof hm, hipMemcpyHostToDevice), "copy mom");
    int32_t slots = 0;
    check(relaysum_num_directed_edges(h, &slots) == RELAYSUM_OK && slots == 4, "4 directed edges");
    for (int32_t s = 0; s < 4; ++s) {
        int32_t src = -1, dst = -1;
        relaysum_directed_edge(h, s, &src, &dst);
        const int32_t want[4][2] = {{0, 1}, {1, 0}, {1, 2}, {2, 1}};
        check(src == want[s][0] && dst == want[s][1], "slot order by source, then destination");
    }
    for (const Round &r : c.rounds) {
        check(relaysum_step(h, x, g, c.beta != 0 ? mom : nullptr, (float)c.lr, (float)c.beta) ==
                  RELAYSUM_OK, "relaysum_step");
        hip_ok(hipDeviceSynchronize(), "round");
        hip_ok(hipMemcpy(hx, x, sizeof hx, hipMemcpyDeviceToHost), "copy x");
        hip_ok(hipMemcpy(hm, mom, sizeof hm, hipMemcpyDeviceToHost), "copy mom");
        int32_t nbar[3], cnt[4];
        check(relaysum_get_counts(h, nbar, cnt) == RELAYSUM_OK, "get_counts");
        for (int i = 0; i < 3; ++i) {
            check(close_to(hx[i], r.x[i]), "x matches the hand-worked value");
            check(nbar[i] == (int32_t)r.nbar[i], "nbar matches");
            if (!r.mom.empty()) check(hm[i] == (float)r.mom[i], "momentum matches exactly");
        }
        for (int32_t s = 0; s < 4; ++s) {
            float m = 0;
            check(relaysum_get_message(h, s, &m) == RELAYSUM_OK, "get_message");
            check(close_to(m, r.m[s]), "message matches the hand-worked value");
            check(cnt[s] == (int32_t)r.c[s], "counter matches");
        }
    }
    int64_t t = -1;
    check(relaysum_round(h, &t) == RELAYSUM_OK && t == (int64_t)c.rounds.size(), "round number");
    // Consensus distance of the last models: (1/3) sum_i (x_i - xbar)^2 and
    // max |x_i - xbar|, in double on the host.
    double mean = 0.0, want = 0.0, want_spread = 0.0;
    for (int i = 0; i < 3; ++i) mean += (double)hx[i];
    mean /= 3.0;
    for (int i = 0; i < 3; ++i) {
        const double e = (double)hx[i] - mean;
        want += e * e;
        want_spread = std::fmax(want_spread, std::fabs(e));
    }
    want /= 3.0;
    double dist = -1.0, spread = -1.0;
    check(relaysum_consensus_distance(h, x, &dist, &spread) == RELAYSUM_OK, "consensus_distance");
    check(std::fabs(dist - want) <= 1e-12 * std::fmax(want, 1e-30) &&
              std::fabs(spread - want_spread) <= 1e-12 * std::fmax(want_spread, 1e-30),
          "consensus distance matches the host's");
    check(relaysum_consensus_distance(h, x, nullptr, nullptr) == RELAYSUM_ERR_INVALID_ARG,
          "consensus_distance needs somewhere to put the distance");
    check(relaysum_destroy(h) == RELAYSUM_OK, "destroy");
    (void)hipFree(x); (void)hipFree(g); (void)hipFree(mom);
}

static void error_codes() {
    relaysum_t *h = (relaysum_t *)0x1;
    const int32_t cycle[6] = {0, 1, 1, 2, 2, 0};
    check(relaysum_create(3, 8, cycle, 3, &h) == RELAYSUM_ERR_NOT_A_TREE && h == nullptr,
          "a cycle is not a tree");
    const int32_t loop[4] = {0, 1, 1, 1};
    check(relaysum_create(3, 8, loop, 2, &h) == RELAYSUM_ERR_NOT_A_TREE, "a self loop is rejected");
    check(relaysum_create(0, 8, nullptr, 0, &h) == RELAYSUM_ERR_INVALID_ARG, "n = 0 is rejected");
    check(relaysum_create(RELAYSUM_MAX_WORKERS + 1, 8, nullptr, RELAYSUM_MAX_WORKERS, &h) ==
              RELAYSUM_ERR_INVALID_ARG,
          "n above RELAYSUM_MAX_WORKERS is rejected");
    check(relaysum_create(2, 8, cycle, 1, nullptr) == RELAYSUM_ERR_INVALID_ARG, "NULL out");
    check(relaysum_destroy(nullptr) == RELAYSUM_OK, "destroy(NULL) is a no-op");
    check(std::strcmp(relaysum_strerror(RELAYSUM_ERR_NOT_A_TREE), "unknown status") != 0,
          "strerror names codes");
    const int32_t chain[6] = {0, 1, 1, 2, 2, 3};
    check(relaysum_create(4, 64, chain, 3, &h) == RELAYSUM_OK, "create a chain of 4");
    float *x;
    hip_ok(hipMalloc((void **)&x, 4 * 64 * sizeof(float)), "hipMalloc");
    relaysum_round_args a;
    std::memset(&a, 0, sizeof a);
    a.update = RELAYSUM_UPDATE_GRAD;
    a.beta1 = 0.9f;
    check(relaysum_step_ex(h, x, x, nullptr, nullptr, &a) == RELAYSUM_ERR_INVALID_ARG,
          "Alg. 4 with momentum is rejected");
    check(std::strlen(relaysum_last_error(h)) > 0, "last_error explains the failure");
    a.update = RELAYSUM_UPDATE_MODEL;
    a.optimizer = RELAYSUM_OPT_ADAM;
    a.adam_step = 0;
    check(relaysum_step_ex(h, x, x, x, x, &a) == RELAYSUM_ERR_INVALID_ARG, "adam_step 0 is rejected");
    check(relaysum_step(h, x, x, nullptr, 0.1f, 0.9f) == RELAYSUM_ERR_INVALID_ARG,
          "momentum without a buffer is rejected");
    check(relaysum_step(h, x, x, nullptr, 0.1f, 0.0f) == RELAYSUM_ERR_INVALID_ARG,
          "x and g in the same buffer are rejected");
    check(relaysum_step(h, x + 64, x, nullptr, 0.1f, 0.0f) == RELAYSUM_ERR_INVALID_ARG,
          "x and g sharing rows are rejected");
    int64_t t = -1;
    relaysum_round(h, &t);
    check(t == 0, "failed calls do not advance the round");
    relaysum_destroy(h);
    (void)hipFree(x);
}

// Section 3: a double-tree handle relays odd coordinates on tree A and even
// ones on tree B, so it equals two single-tree handles on those coordinates.
static void double_trees() {
    const int n = 5, d = 12, dh = d / 2;
    const int32_t ea[8] = {0, 1, 1, 2, 2, 3, 3, 4};     // chain
    const int32_t eb[8] = {2, 0, 2, 1, 2, 3, 2, 4};     // star around worker 2
    relaysum_t *hd = nullptr, *ha = nullptr, *hb = nullptr;
    check(relaysum_create_double(n, d, ea, eb, 4, &hd) == RELAYSUM_OK, "create double trees");
    check(relaysum_create(n, dh, ea, 4, &ha) == RELAYSUM_OK, "create tree A");
    check(relaysum_create(n, dh, eb, 4, &hb) == RELAYSUM_OK, "create tree B");
    int32_t trees = 0, slots = 0;
    int64_t len = 0;
    relaysum_num_trees(hd, &trees);
    relaysum_num_directed_edges(hd, &slots);
    relaysum_message_length(hd, 0, &len);
    check(trees == 2 && slots == 16 && len == dh, "double-tree handle shape");
    std::vector<float> hx(n * d), hg(n * d), ax(n * dh), ag(n * dh), bx(n * dh), bg(n * dh);
    for (int i = 0; i < n * d; ++i) {
        hx[i] = std::sin(0.37f * (float)i);
        hg[i] = std::cos(0.11f * (float)i);
    }
    for (int i = 0; i < n; ++i)
        for (int c = 0; c < d; ++c) {
            std::vector<float> &dx = (c & 1) ? ax : bx, &dg = (c & 1) ? ag : bg;
            dx[i * dh + c / 2] = hx[i * d + c];
            dg[i * dh + c / 2] = hg[i * d + c];
        }
    float *x, *g, *m, *xa, *ga, *ma, *xb, *gb, *mb;
    const size_t full = n * d * sizeof(float), half = n * dh * sizeof(float);
    hip_ok(hipMalloc((void **)&x, full), "hipMalloc"); hip_ok(hipMalloc((void **)&g, full), "hipMalloc");
    hip_ok(hipMalloc((void **)&m, full), "hipMalloc"); hip_ok(hipMalloc((void **)&xa, half), "hipMalloc");
    hip_ok(hipMalloc((void **)&ga, half), "hipMalloc"); hip_ok(hipMalloc((void **)&ma, half), "hipMalloc");
    hip_ok(hipMalloc((void **)&xb, half), "hipMalloc"); hip_ok(hipMalloc((void **)&gb, half), "hipMalloc");
    hip_ok(hipMalloc((void **)&mb, half), "hipMalloc");
    hip_ok(hipMemcpy(x, hx.data(), full, hipMemcpyHostToDevice), "copy");
    hip_ok(hipMemcpy(g, hg.data(), full, hipMemcpyHostToDevice), "copy");
    hip_ok(hipMemcpy(xa, ax.data(), half, hipMemcpyHostToDevice), "copy");
    hip_ok(hipMemcpy(ga, ag.data(), half, hipMemcpyHostToDevice), "copy");
    hip_ok(hipMemcpy(xb, bx.data(), half, hipMemcpyHostToDevice), "copy");
    hip_ok(hipMemcpy(gb, bg.data(), half, hipMemcpyHostToDevice), "copy");
    hip_ok(hipMemset(m, 0, full), "memset"); hip_ok(hipMemset(ma, 0, half), "memset");
    hip_ok(hipMemset(mb, 0, half), "memset");
    for (int r = 0; r < 6; ++r) {
        check(relaysum_step(hd, x, g, m, 0.1f, 0.9f) == RELAYSUM_OK, "double-tree step");
        check(relaysum_step(ha, xa, ga, ma, 0.1f, 0.9f) == RELAYSUM_OK, "tree A step");
        check(relaysum_step(hb, xb, gb, mb, 0.1f, 0.9f) == RELAYSUM_OK, "tree B step");
    }
    hip_ok(hipDeviceSynchronize(), "rounds");
    hip_ok(hipMemcpy(hx.data(), x, full, hipMemcpyDeviceToHost), "copy");
    hip_ok(hipMemcpy(ax.data(), xa, half, hipMemcpyDeviceToHost), "copy");
    hip_ok(hipMemcpy(bx.data(), xb, half, hipMemcpyDeviceToHost), "copy");
    int same = 1;
    for (int i = 0; i < n; ++i)
        for (int c = 0; c < d; ++c) {
            const float want = ((c & 1) ? ax : bx)[i * dh + c / 2];
            same &= std::memcmp(&hx[i * d + c], &want, sizeof(float)) == 0;
        }
    check(same, "double trees equal the two single trees bit for bit");
    relaysum_destroy(hd); relaysum_destroy(ha); relaysum_destroy(hb);
    for (float *p : {x, g, m, xa, ga, ma, xb, gb, mb}) (void)hipFree(p);
}

// A snapshot taken after 3 of 6 rounds and loaded into a fresh handle
// resumes the run: its last 3 rounds give the models and messages of 6
// straight rounds, bit for bit; a snapshot of another tree is rejected.
static void snapshots() {
    const int n = 6, d = 40;
    const int32_t edges[10] = {0, 1, 1, 2, 1, 3, 3, 4, 3, 5};
    const int32_t other[10] = {0, 1, 1, 2, 2, 3, 3, 4, 4, 5};
    relaysum_t *a = nullptr, *b = nullptr, *c = nullptr, *o = nullptr;
    check(relaysum_create(n, d, edges, 5, &a) == RELAYSUM_OK, "create (straight run)");
    check(relaysum_create(n, d, edges, 5, &b) == RELAYSUM_OK, "create (saved run)");
    check(relaysum_create(n, d, edges, 5, &c) == RELAYSUM_OK, "create (resumed run)");
    check(relaysum_create(n, d, other, 5, &o) == RELAYSUM_OK, "create (other tree)");
    const size_t bytes = (size_t)n * d * sizeof(float);
    std::vector<float> hx(n * d), hg(n * d);
    for (int i = 0; i < n * d; ++i) hx[i] = std::sin(0.23f * (float)i);
    float *xa, *ma, *xb, *mb, *g;
    for (float **p : {&xa, &ma, &xb, &mb, &g}) hip_ok(hipMalloc((void **)p, bytes), "hipMalloc");
    hip_ok(hipMemcpy(xa, hx.data(), bytes, hipMemcpyHostToDevice), "copy");
    hip_ok(hipMemcpy(xb, hx.data(), bytes, hipMemcpyHostToDevice), "copy");
    hip_ok(hipMemset(ma, 0, bytes), "memset");
    hip_ok(hipMemset(mb, 0, bytes), "memset");
    auto grad = [&](int r) {
        for (int i = 0; i < n * d; ++i) hg[i] = std::cos(0.07f * (float)(i + 31 * r));
        hip_ok(hipMemcpy(g, hg.data(), bytes, hipMemcpyHostToDevice), "copy");
    };
    for (int r = 0; r < 6; ++r) {
        grad(r);
        check(relaysum_step(a, xa, g, ma, 0.1f, 0.9f) == RELAYSUM_OK, "straight step");
        hip_ok(hipDeviceSynchronize(), "round");
    }
    for (int r = 0; r < 3; ++r) {
        grad(r);
        check(relaysum_step(b, xb, g, mb, 0.1f, 0.9f) == RELAYSUM_OK, "step before the snapshot");
        hip_ok(hipDeviceSynchronize(), "round");
    }
    size_t size = 0;
    check(relaysum_state_size(b, &size) == RELAYSUM_OK && size > 0, "state_size");
    std::vector<unsigned char> snap(size);
    check(relaysum_save_state(b, snap.data(), size - 1) == RELAYSUM_ERR_INVALID_ARG,
          "save_state rejects a short buffer");
    check(relaysum_save_state(b, snap.data(), size) == RELAYSUM_OK, "save_state");
    check(relaysum_load_state(o, snap.data(), size) == RELAYSUM_ERR_INVALID_ARG,
          "load_state rejects a snapshot of another tree");
    check(relaysum_load_state(c, snap.data(), size) == RELAYSUM_OK, "load_state");
    int64_t t = 0;
    relaysum_round(c, &t);
    check(t == 3, "the loaded round number");
    for (int r = 3; r < 6; ++r) {
        grad(r);
        check(relaysum_step(c, xb, g, mb, 0.1f, 0.9f) == RELAYSUM_OK, "step after loading");
        hip_ok(hipDeviceSynchronize(), "round");
    }
    std::vector<float> ya(n * d), yb(n * d), ma_h(d), mb_h(d);
    hip_ok(hipMemcpy(ya.data(), xa, bytes, hipMemcpyDeviceToHost), "copy");
    hip_ok(hipMemcpy(yb.data(), xb, bytes, hipMemcpyDeviceToHost), "copy");
    int same = std::memcmp(ya.data(), yb.data(), bytes) == 0;
    for (int s = 0; s < 10; ++s) {
        check(relaysum_get_message(a, s, ma_h.data()) == RELAYSUM_OK &&
                  relaysum_get_message(c, s, mb_h.data()) == RELAYSUM_OK, "get_message");
        same &= std::memcmp(ma_h.data(), mb_h.data(), d * sizeof(float)) == 0;
    }
    check(same, "resumed run equals the straight run bit for bit");
    for (relaysum_t *h : {a, b, c, o}) relaysum_destroy(h);
    for (float *p : {xa, ma, xb, mb, g}) (void)hipFree(p);
}

int main(int argc, char **argv) {
    if (argc < 2) {
        std::printf("usage: %s <chain3_alg1_hand_worked.txt>\n", argv[0]);
        return 2;
    }
    hand_worked_chain(argv[1], "lr0");
    hand_worked_chain(argv[1], "nesterov");
    error_codes();
    double_trees();
    snapshots();
    std::printf("relaysum C ABI check: %d of %d checks passed\n", g_checks - g_failed, g_checks);
    return g_failed == 0 ? 0 : 1;
}
