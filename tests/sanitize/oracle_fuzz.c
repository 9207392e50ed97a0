/*
 * Host check of the C oracle (oracle/dtree_oracle.c) built with AddressSanitizer and
 * UndefinedBehaviorSanitizer: random full trees and forests over record matrices with
 * row strides above the feature count, special values, no records, and corrupted trees
 * (which must be reported, not walked out of bounds).  Labels must agree between the
 * single-tree entry points and a one-tree forest.  Usage: oracle_fuzz SEED TREES
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

typedef struct {
    int32_t feature;
    float threshold;
    int32_t left;
    int32_t cls;
} oracle_node;

int oracle_tree_leaves(const oracle_node *, int32_t, int32_t, const float *, int64_t, int64_t,
                       int32_t *);
int oracle_tree_classes(const oracle_node *, int32_t, int32_t, const float *, int64_t, int64_t,
                        int32_t *);
int oracle_forest_classes(const oracle_node *, const int32_t *, int32_t, int32_t, int32_t,
                          const float *, int64_t, int64_t, int32_t *);

static uint64_t state;
static uint64_t next_u64(void) {   /* splitmix64 */
    uint64_t z = (state += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}
static int below(int n) { return (int)(next_u64() % (uint64_t)n); }
static float value(void) {
    switch (below(10)) {
        case 0: return NAN;
        case 1: return INFINITY;
        case 2: return -INFINITY;
        case 3: return -0.0f;
        default: return (float)(next_u64() >> 40) / (float)(1 << 24);
    }
}

/* Complete tree of the given depth in breadth-first layout: node i's children are 2i+1
 * and 2i+2 (depth 0: one leaf). */
static int complete_tree(oracle_node *t, int depth, int F, int C) {
    const int n = (1 << (depth + 1)) - 1;
    for (int i = 0; i < n; ++i) {
        if (2 * i + 1 < n) {
            t[i].feature = below(F); t[i].threshold = value(); t[i].left = 2 * i + 1; t[i].cls = -1;
        } else {
            t[i].feature = 0; t[i].threshold = 0.0f; t[i].left = -1; t[i].cls = below(C);
        }
    }
    return n;
}

int main(int argc, char **argv) {
    state = argc > 1 ? strtoull(argv[1], NULL, 10) : 1;
    const int trees = argc > 2 ? atoi(argv[2]) : 200;
    for (int it = 0; it < trees; ++it) {
        const int F = 1 + below(33), C = 1 + below(40), depth = below(11);
        const int64_t n = below(300), ld = F + below(5);
        oracle_node *t = malloc(sizeof(oracle_node) * (size_t)((1 << 12)));
        float *x = malloc(sizeof(float) * (size_t)((n + 1) * ld));   /* >= one row */
        int32_t *a = malloc(sizeof(int32_t) * (size_t)(n + 1));
        int32_t *b = malloc(sizeof(int32_t) * (size_t)(n + 1));
        int32_t *leaf = malloc(sizeof(int32_t) * (size_t)(n + 1));
        if (!t || !x || !a || !b || !leaf) return 2;
        const int nn = complete_tree(t, depth, F, C);
        for (int64_t i = 0; i < (n + 1) * ld; ++i) x[i] = value();
        int32_t offsets[2] = {0, nn};
        if (oracle_tree_classes(t, nn, F, x, n, ld, a) != 0) { fprintf(stderr, "FAIL classes %d\n", it); return 1; }
        if (oracle_tree_leaves(t, nn, F, x, n, ld, leaf) != 0) { fprintf(stderr, "FAIL leaves %d\n", it); return 1; }
        if (oracle_forest_classes(t, offsets, 1, F, C, x, n, ld, b) != 0) { fprintf(stderr, "FAIL forest %d\n", it); return 1; }
        for (int64_t s = 0; s < n; ++s)
            if (a[s] != b[s] || a[s] != t[leaf[s]].cls) { fprintf(stderr, "FAIL agree %d\n", it); return 1; }
        if (depth > 0) {
            /* corrupted roots, on one row: a right child past the end and a feature out of
             * range must be reported; a left edge back to the root (a cycle for records
             * that go left) must end, reported or not */
            for (int kind = 0; kind < 3; ++kind) {
                const oracle_node save = t[0];
                if (kind == 0) t[0].left = nn - 1;
                else if (kind == 1) t[0].left = 0;
                else t[0].feature = F;
                const int rc = oracle_tree_classes(t, nn, F, x, 1, ld, a);
                if (rc == 0 && kind != 1) { fprintf(stderr, "FAIL corrupt accepted %d %d\n", it, kind); return 1; }
                t[0] = save;
            }
        }
        free(t); free(x); free(a); free(b); free(leaf);
    }
    printf("ok\n");
    return 0;
}
