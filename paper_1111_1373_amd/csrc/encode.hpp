// Host-side tree validation and window encoding shared by both GPU decompositions.
//
// A window is a block of at most D levels of the tree, rooted at a decision node and
// embedded in a complete binary heap stored 1-based: slot p in [1, 2^D) holds heap node p
// (children 2p and 2p+1, so the two children of a node are one aligned 16-byte pair), and
// slot 0 is padding.  Leaving the window at bottom position 2^D + e is exit e.
// This is the "window" of Section 6 of the paper (evaluate a few levels, then continue
// from the node reached), and it gives the speculative decomposition its fixed lane map
// (the processor-node map of Procedure 5): lane h of a record's lane group evaluates
// slot h.  Slots that hold no decision node (below a leaf that ends the path early)
// always send the record right, so a leaf met above the bottom is recorded at the exit
// reached by going right from it; this plays the role of Procedure 5's static leaf
// paths.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

#include "dtree.h"

namespace dtree {

constexpr int kMaxNodes = 1 << 24;
constexpr int kMaxWindowDepth = 16;
constexpr int kMaxSpecWindowDepth = 6;
// Default speculative window depth: 4-lane record groups measured fastest on MI355X (the
// paper's 16-lane groups are depth 4).
constexpr int kDefaultSpecWindowDepth = 2;

// Parsed, validated tree.
struct TreeShape {
    int32_t n_nodes = 0, n_internal = 0, n_leaves = 0, depth = 0;
    std::vector<int32_t> node_depth;   // edges from the root
};

// Validates the layout rules of dtree.h.  Returns DT_OK or an error with `msg` set.
dt_status validate_tree(const dt_node *nodes, int32_t n_nodes, int32_t n_features,
                        int32_t n_classes, TreeShape *shape, std::string *msg);

// Window encoding (see dt_encode_windows in dtree.h).  Slot-major arrays of
// n_windows * 2^depth entries.
struct WindowTables {
    int32_t depth = 0;        // D
    int32_t slots = 0;        // S = 2^D
    int32_t n_windows = 0;
    int32_t levels = 0;       // windows on the longest root-to-leaf path
    int32_t first_depth = 0;  // decision levels of window 0 (d0 <= D; the others have D)
    std::vector<int32_t> feature;
    std::vector<float> threshold;
    std::vector<int32_t> exit_class;
    std::vector<int32_t> exit_leaf;
};

// Slot words of the windows for narrow records (fp16, bf16, uint8): feature index << 16 |
// key, where the key is the threshold moved onto the record type's grid, rounded up: the
// smallest value of the type (as its bits) not below t, and for uint8 the integer ceiling
// of t clamped to 0..256.  No representable record value lies in [t, key), so a stored
// element x satisfies x < key exactly when its widened value is below t.  A NaN threshold
// sends every record right (key NaN, or 0 for uint8).  One word per slot, slot-major.
uint32_t narrow_key(float t, dt_dtype type);
void build_narrow_slots(const WindowTables &wt, dt_dtype type, std::vector<uint32_t> *out);

// Depth d0 of the first window for window depth D: windows are rooted at tree depth 0 and
// at depths d0, d0 + D, d0 + 2D, ...  d0 is D, or the depth that fills the deepest level of
// windows when that needs fewer windows.
int first_window_depth(const dt_node *nodes, const TreeShape &shape, int depth);

// Number of windows, and window levels on the longest path, for window depth D (without
// building them).
int64_t count_windows(const dt_node *nodes, const TreeShape &shape, int depth);
int32_t count_levels(const dt_node *nodes, const TreeShape &shape, int depth);

void build_windows(const dt_node *nodes, const TreeShape &shape, int depth, WindowTables *out);

// Bytes a workgroup stages in LDS for a table of n_windows windows of 2^depth slots:
// one 8-byte (threshold, feature) pair and one 4-byte exit per slot.
inline int64_t table_bytes(int64_t n_windows, int depth) {
    return n_windows * (int64_t(1) << depth) * 12;
}

// LDS bytes of a gfx950 workgroup, and the most LDS the default data windows may take.
constexpr int64_t kLdsBytes = 160 * 1024;
constexpr int64_t kDataTableBudget = 48 * 1024;

// Table bytes the default data window depth may use for records of n_features: at most
// kDataTableBudget, and room left for two fp32 record tiles.
int64_t data_table_budget(int32_t n_features);

// Library's default window depths (see dt_tree_options in dtree.h).  Data: the fewest
// window levels among the depths whose tables fit max_bytes (ties: smaller tables), or the
// smallest tables if none fits.
int choose_data_window_depth(const dt_node *nodes, const TreeShape &shape, int64_t max_bytes);
int choose_spec_window_depth(const TreeShape &shape);

}  // namespace dtree
