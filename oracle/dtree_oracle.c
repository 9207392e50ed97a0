/*
 * Serial CPU oracle for classification-tree evaluation.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the package smoke check and the
 * benchmark's CPU-baseline leg may load this code.  It shares no source, header, table
 * or helper with the GPU library, and the GPU library never calls it.
 *
 * What it computes (Spencer, "Speculative Parallel Evaluation of Classification Trees on
 * GPGPU Compute Engines"):
 *   - Section 2.1 / Section 3.1 problem statement: every record R is assigned the class
 *     of the leaf reached by recursive evaluation from the root n_0.
 *   - The decision at node n compares attribute r_{a_n} with threshold t_n.  This library
 *     uses the comparison "x < t goes to the left child, otherwise to the right child"
 *     (so x == t and NaN go right).  The paper writes the complementary form with
 *     "r <= t goes left"; a tree in that form converts by replacing every threshold t by
 *     the next float above t.
 *   - Trees arrive in the breadth-first array of Procedure 1: a node stores its feature,
 *     threshold, the index of its left child (the right child is the next index) and a
 *     class, with cls < 0 standing for the paper's "no class" of a decision node.
 *   - Forests (Section 1, Sharp's concatenated trees): each tree votes for its class;
 *     the label is the class with most votes, ties going to the smallest class id.
 *
 * This is written as the plain definition: an explicit if/else walk from the root with
 * two named children.  It does not use Procedure 2's "child + predicate" arithmetic,
 * leaf self-loops, windows or bit masks.  Compile without -ffast-math so that the
 * comparison keeps IEEE semantics (NaN compares false, denormals are not flushed).
 */
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>

typedef struct {
    int32_t feature;    /* 0-based attribute index a_n - 1; unused for leaves     */
    float threshold;    /* t_n; unused for leaves                                  */
    int32_t left;       /* index of the left child; right child is left + 1       */
    int32_t cls;        /* class c_n of a leaf; negative for a decision node      */
} oracle_node;

enum { ORACLE_OK = 0, ORACLE_BAD_TREE = -1, ORACLE_BAD_ARG = -2 };

/* Leaf reached by one record: recursive evaluation from the root (Section 3.1). */
static int32_t leaf_of_record(const oracle_node *nodes, int32_t n_nodes, int32_t n_features,
                              const float *row)
{
    int32_t i = 0;
    int32_t steps = 0;
    while (nodes[i].cls < 0) {
        const oracle_node *n = &nodes[i];
        if (n->feature < 0 || n->feature >= n_features) return -1;
        if (n->left < 0 || n->left + 1 >= n_nodes) return -1;
        float x = row[n->feature];
        int32_t left_child = n->left;
        int32_t right_child = n->left + 1;
        if (x < n->threshold) {
            i = left_child;
        } else {
            i = right_child;
        }
        if (++steps > n_nodes) return -1;  /* a cycle: not a tree */
    }
    return i;
}

/* leaf[s] = index of the leaf reached by record s.  Returns ORACLE_OK or an error. */
int oracle_tree_leaves(const oracle_node *nodes, int32_t n_nodes, int32_t n_features,
                       const float *x, int64_t n, int64_t ld, int32_t *leaf)
{
    if (!nodes || n_nodes <= 0 || n < 0 || ld < n_features || (n > 0 && (!x || !leaf)))
        return ORACLE_BAD_ARG;
    for (int64_t s = 0; s < n; ++s) {
        int32_t l = leaf_of_record(nodes, n_nodes, n_features, x + s * ld);
        if (l < 0) return ORACLE_BAD_TREE;
        leaf[s] = l;
    }
    return ORACLE_OK;
}

/* label[s] = class of the leaf reached by record s (Procedure 2's output). */
int oracle_tree_classes(const oracle_node *nodes, int32_t n_nodes, int32_t n_features,
                        const float *x, int64_t n, int64_t ld, int32_t *label)
{
    if (!nodes || n_nodes <= 0 || n < 0 || ld < n_features || (n > 0 && (!x || !label)))
        return ORACLE_BAD_ARG;
    for (int64_t s = 0; s < n; ++s) {
        int32_t l = leaf_of_record(nodes, n_nodes, n_features, x + s * ld);
        if (l < 0) return ORACLE_BAD_TREE;
        label[s] = nodes[l].cls;
    }
    return ORACLE_OK;
}

/*
 * Forest majority vote.  Tree k occupies nodes[offsets[k] .. offsets[k+1]) and its child
 * indices are local to that range.  label[s] = argmax_c votes[c], smallest c on ties.
 */
int oracle_forest_classes(const oracle_node *nodes, const int32_t *offsets, int32_t n_trees,
                          int32_t n_features, int32_t n_classes, const float *x, int64_t n,
                          int64_t ld, int32_t *label)
{
    if (!nodes || !offsets || n_trees <= 0 || n_classes <= 0 || n < 0 || ld < n_features ||
        (n > 0 && (!x || !label)))
        return ORACLE_BAD_ARG;
    int32_t *votes = (int32_t *)calloc((size_t)n_classes, sizeof(int32_t));
    if (!votes) return ORACLE_BAD_ARG;
    int rc = ORACLE_OK;
    for (int64_t s = 0; s < n && rc == ORACLE_OK; ++s) {
        const float *row = x + s * ld;
        for (int32_t c = 0; c < n_classes; ++c) votes[c] = 0;
        for (int32_t k = 0; k < n_trees; ++k) {
            const oracle_node *tree = nodes + offsets[k];
            int32_t size = offsets[k + 1] - offsets[k];
            int32_t l = leaf_of_record(tree, size, n_features, row);
            if (l < 0) { rc = ORACLE_BAD_TREE; break; }
            int32_t c = tree[l].cls;
            if (c >= n_classes) { rc = ORACLE_BAD_TREE; break; }
            votes[c] += 1;
        }
        int32_t best = 0;
        for (int32_t c = 1; c < n_classes; ++c)
            if (votes[c] > votes[best]) best = c;   /* strict: ties keep the smaller id */
        label[s] = best;
    }
    free(votes);
    return rc;
}
