// Host check of the tree validation and window encoder (encode.cpp) built with
// AddressSanitizer and UndefinedBehaviorSanitizer.  Random full trees in the breadth-first
// layout of Procedure 1 are encoded at every window depth 1..8; walking each record
// through the window tables (D heap steps per window, then the exit) must reach the leaf
// a direct walk of the tree reaches.  Corrupted arrays must be rejected, not crash.
// Usage: encode_fuzz SEED TREES
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <limits>
#include <string>
#include <vector>

#include "encode.hpp"

namespace {

uint64_t g_state;
uint64_t next_u64() {   // splitmix64
    uint64_t z = (g_state += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}
int below(int n) { return int(next_u64() % uint64_t(n)); }
float unit() { return float(next_u64() >> 40) / float(1 << 24); }

float special_or_unit() {
    switch (below(12)) {
        case 0: return std::numeric_limits<float>::quiet_NaN();
        case 1: return std::numeric_limits<float>::infinity();
        case 2: return -std::numeric_limits<float>::infinity();
        case 3: return -0.0f;
        case 4: return std::numeric_limits<float>::denorm_min();
        default: return unit();
    }
}

// Random full binary tree with n_int decision nodes (split random leaves), renumbered
// breadth-first so that every node's right child directly follows its left child.
std::vector<dt_node> random_tree(int n_int, int F, int C) {
    struct Kids { int l = -1; };
    std::vector<Kids> t(1);
    std::vector<int> leaves{0};
    for (int k = 0; k < n_int; ++k) {
        const int pick = below(int(leaves.size()));
        const int v = leaves[size_t(pick)];
        leaves[size_t(pick)] = leaves.back();
        leaves.pop_back();
        const int a = int(t.size());
        t.resize(t.size() + 2);
        t[size_t(v)].l = a;
        leaves.push_back(a);
        leaves.push_back(a + 1);
    }
    std::vector<int> order{0}, id(t.size());
    for (size_t h = 0; h < order.size(); ++h) {
        const int v = order[h];
        id[size_t(v)] = int(h);
        if (t[size_t(v)].l >= 0) {
            order.push_back(t[size_t(v)].l);
            order.push_back(t[size_t(v)].l + 1);
        }
    }
    std::vector<dt_node> out(order.size());
    for (size_t h = 0; h < order.size(); ++h) {
        const int v = order[h];
        if (t[size_t(v)].l >= 0)
            out[h] = dt_node{below(F), special_or_unit(), id[size_t(t[size_t(v)].l)], -1};
        else
            out[h] = dt_node{0, 0.0f, -1, below(C)};
    }
    return out;
}

int direct_leaf(const std::vector<dt_node> &t, const float *x) {
    int i = 0;
    while (t[size_t(i)].cls < 0)
        i = x[t[size_t(i)].feature] < t[size_t(i)].threshold ? t[size_t(i)].left
                                                              : t[size_t(i)].left + 1;
    return i;
}

int window_leaf(const dtree::WindowTables &wt, const float *x) {
    int w = 0;
    for (int level = 0; level < wt.levels; ++level) {
        int p = 1;
        for (int k = 0; k < wt.depth; ++k) {
            const size_t s = size_t(w) * size_t(wt.slots) + size_t(p);
            p = 2 * p + int(!(x[wt.feature[s]] < wt.threshold[s]));
        }
        const int code = wt.exit_leaf[size_t(w) * size_t(wt.slots) + size_t(p - wt.slots)];
        if (code < 0) return -code - 1;
        if (code >= wt.n_windows) return -2;
        w = code;
    }
    return -3;   // more windows on a path than `levels`
}

int fail(const char *what, int a, int b) {
    std::fprintf(stderr, "FAIL %s (%d, %d)\n", what, a, b);
    return 1;
}

}  // namespace

int main(int argc, char **argv) {
    g_state = argc > 1 ? std::strtoull(argv[1], nullptr, 10) : 1;
    const int trees = argc > 2 ? std::atoi(argv[2]) : 200;
    const int sizes[] = {0, 1, 2, 3, 7, 15, 40, 63, 64, 200, 1000, 3000};
    long checked = 0;
    for (int it = 0; it < trees; ++it) {
        const int F = 1 + below(40), C = 1 + below(300);
        const int n_int = sizes[below(int(sizeof(sizes) / sizeof(sizes[0])))];
        const std::vector<dt_node> t = random_tree(n_int, F, C);
        dtree::TreeShape shape;
        std::string msg;
        if (dtree::validate_tree(t.data(), int32_t(t.size()), F, C, &shape, &msg) != DT_OK)
            return fail("valid tree rejected", it, n_int);
        std::vector<float> x(size_t(64) * size_t(F + 1));
        for (float &v : x) v = special_or_unit();
        for (int r = 0; r < 64 && n_int > 0; ++r) {   // ties on some decision node
            const int node = below(int(t.size()));
            if (t[size_t(node)].cls < 0)
                x[size_t(r) * size_t(F + 1) + size_t(t[size_t(node)].feature)] =
                    t[size_t(node)].threshold;
        }
        for (int D = 1; D <= 8; ++D) {
            dtree::WindowTables wt;
            dtree::build_windows(t.data(), shape, D, &wt);
            if (wt.n_windows != dtree::count_windows(t.data(), shape, D))
                return fail("window count", it, D);
            if (wt.levels != dtree::count_levels(t.data(), shape, D))
                return fail("window levels", it, D);
            for (int32_t e : wt.exit_class)
                if (e < -C || e >= wt.n_windows) return fail("exit code range", it, e);
            for (int r = 0; r < 64; ++r) {
                const float *row = x.data() + size_t(r) * size_t(F + 1);
                const int a = direct_leaf(t, row), b = window_leaf(wt, row);
                if (a != b) return fail("window walk leaf", a, b);
                ++checked;
            }
        }
        // corrupted copies: validation must reject them
        if (n_int > 0) {
            for (int kind = 0; kind < 5; ++kind) {
                std::vector<dt_node> bad = t;
                int node = below(int(bad.size()));
                while (bad[size_t(node)].cls >= 0) node = below(int(bad.size()));
                switch (kind) {
                    case 0: bad[size_t(node)].left = node; break;                      // back edge
                    case 1: bad[size_t(node)].left = int(bad.size()) - 1; break;       // right out of range
                    case 2: bad[size_t(node)].feature = F; break;
                    case 3: bad[size_t(bad.size()) - 1].cls = C; break;
                    default: bad.pop_back(); break;                                    // truncated
                }
                dtree::TreeShape s2;
                if (dtree::validate_tree(bad.data(), int32_t(bad.size()), F, C, &s2, &msg) == DT_OK)
                    return fail("corrupt tree accepted", it, kind);
            }
        }
        for (int k = 0; k < 64; ++k) {   // narrow threshold keys of arbitrary floats
            const float v = k % 2 ? special_or_unit() : (unit() - 0.5f) * 1e6f;
            if (dtree::narrow_key(v, DT_U8) > 256u) return fail("uint8 key range", it, k);
            (void)dtree::narrow_key(v, DT_F16);
            (void)dtree::narrow_key(v, DT_BF16);
        }
    }
    std::printf("ok %ld walks\n", checked);
    return 0;
}
