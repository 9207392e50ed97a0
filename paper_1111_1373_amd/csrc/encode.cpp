// Tree validation and window encoding (host only).  See encode.hpp.
#include "encode.hpp"

#include <algorithm>
#include <cmath>
#include <cstring>
#include <limits>

namespace dtree {

dt_status validate_tree(const dt_node *nodes, int32_t n_nodes, int32_t n_features,
                        int32_t n_classes, TreeShape *shape, std::string *msg) {
    if (!nodes) { *msg = "nodes is NULL"; return DT_ERR_INVALID_ARG; }
    if (n_nodes < 1) { *msg = "n_nodes must be >= 1"; return DT_ERR_INVALID_ARG; }
    if (n_features < 1) { *msg = "n_features must be >= 1"; return DT_ERR_INVALID_ARG; }
    if (n_classes < 1) { *msg = "n_classes must be >= 1"; return DT_ERR_INVALID_ARG; }
    if (n_nodes > kMaxNodes) {
        *msg = "trees are limited to 2^24 nodes";
        return DT_ERR_UNSUPPORTED;
    }
    std::vector<int32_t> parent(n_nodes, -1);
    int32_t n_internal = 0;
    for (int32_t i = 0; i < n_nodes; ++i) {
        const dt_node &n = nodes[i];
        if (n.cls == -1) {
            ++n_internal;
            if (n.feature < 0 || n.feature >= n_features) {
                *msg = "node " + std::to_string(i) + ": feature " + std::to_string(n.feature) +
                       " outside [0, n_features)";
                return DT_ERR_INVALID_TREE;
            }
            if (n.left <= i || n.left >= n_nodes - 1) {
                *msg = "node " + std::to_string(i) + ": left child " + std::to_string(n.left) +
                       " must satisfy i < left and left + 1 < n_nodes";
                return DT_ERR_INVALID_TREE;
            }
            for (int32_t c = n.left; c <= n.left + 1; ++c) {
                if (parent[c] != -1) {
                    *msg = "node " + std::to_string(c) + " has two parents (" +
                           std::to_string(parent[c]) + " and " + std::to_string(i) + ")";
                    return DT_ERR_INVALID_TREE;
                }
                parent[c] = i;
            }
        } else if (n.cls < 0 || n.cls >= n_classes) {
            *msg = "node " + std::to_string(i) + ": class " + std::to_string(n.cls) +
                   " outside [0, n_classes) (use -1 for a decision node)";
            return DT_ERR_INVALID_TREE;
        }
    }
    // With forward edges and single parents every node 1..n-1 hangs below the root; a
    // full binary tree then has exactly n_nodes = 2 * n_internal + 1.
    for (int32_t i = 1; i < n_nodes; ++i) {
        if (parent[i] < 0) {
            *msg = "node " + std::to_string(i) + " has no parent";
            return DT_ERR_INVALID_TREE;
        }
    }
    if (n_nodes != 2 * n_internal + 1) {
        *msg = "not a full binary tree";
        return DT_ERR_INVALID_TREE;
    }
    shape->n_nodes = n_nodes;
    shape->n_internal = n_internal;
    shape->n_leaves = n_nodes - n_internal;
    shape->node_depth.assign(n_nodes, 0);
    int32_t depth = 0;
    for (int32_t i = 1; i < n_nodes; ++i) {   // parent index < child index
        shape->node_depth[i] = shape->node_depth[parent[i]] + 1;
        depth = std::max(depth, shape->node_depth[i]);
    }
    shape->depth = depth;
    return DT_OK;
}

namespace {

// Window roots for window depth D and first-window depth d0: the root and every decision
// node at depth d0 + m D (m >= 0).
int64_t count_roots(const dt_node *nodes, const TreeShape &shape, int depth, int first) {
    int64_t n = 1;
    for (int32_t i = 1; i < shape.n_nodes; ++i) {
        const int32_t d = shape.node_depth[i];
        if (nodes[i].cls == -1 && d >= first && (d - first) % depth == 0) ++n;
    }
    return n;
}

}  // namespace

int first_window_depth(const dt_node *nodes, const TreeShape &shape, int depth) {
    // The window levels a record passes through are ceil(depth_of_tree / D) either way;
    // rooting the windows at d0, d0 + D, ... with d0 = depth_of_tree - D (levels - 1)
    // fills the deepest level of windows instead of the first, which often needs far fewer
    // windows (a complete depth-12 tree at D = 5: 1 + 4 + 128 against 1 + 32 + 1024).
    if (shape.depth <= depth) return depth;
    const int levels = (shape.depth + depth - 1) / depth;
    const int shallow = shape.depth - depth * (levels - 1);
    if (shallow == depth) return depth;
    return count_roots(nodes, shape, depth, shallow) < count_roots(nodes, shape, depth, depth)
               ? shallow
               : depth;
}

int64_t count_windows(const dt_node *nodes, const TreeShape &shape, int depth) {
    return count_roots(nodes, shape, depth, first_window_depth(nodes, shape, depth));
}

int32_t count_levels(const dt_node *nodes, const TreeShape &shape, int depth) {
    // a leaf at depth d <= d0 is reached in window level 0, a deeper one in level
    // ceil((d - d0) / D)
    const int first = first_window_depth(nodes, shape, depth);
    if (shape.depth <= first) return 1;
    return 1 + (shape.depth - first + depth - 1) / depth;
}

void build_windows(const dt_node *nodes, const TreeShape &shape, int depth, WindowTables *out) {
    const int32_t S = 1 << depth;
    const float neg_inf = -std::numeric_limits<float>::infinity();
    out->depth = depth;
    out->slots = S;
    const int first = first_window_depth(nodes, shape, depth);
    out->first_depth = first;
    out->levels = count_levels(nodes, shape, depth);
    const int64_t nw = count_windows(nodes, shape, depth);
    out->n_windows = int32_t(nw);
    out->feature.assign(size_t(nw) * S, 0);
    out->threshold.assign(size_t(nw) * S, neg_inf);
    out->exit_class.assign(size_t(nw) * S, -1);
    out->exit_leaf.assign(size_t(nw) * S, -1);

    std::vector<int32_t> roots;
    roots.reserve(size_t(nw));
    roots.push_back(0);
    std::vector<int32_t> slot_node(size_t(S), -1);
    for (size_t w = 0; w < roots.size(); ++w) {
        std::fill(slot_node.begin(), slot_node.end(), -1);
        slot_node[0] = roots[w];
        const size_t base = w * size_t(S);
        // decision levels of this window: d0 for window 0, D for the others; a shallower
        // window's slots below its last level stay always-right padding
        const int dw = w == 0 ? first : depth;
        // h is the 0-based heap index of the working array (stored at slot h + 1).
        // Unreachable exits end the walk like any leaf would; they stay -1.
        for (int32_t h = 0; h < S - 1; ++h) {
            const int32_t n = slot_node[size_t(h)];
            if (n < 0) continue;                          // below an early leaf
            const int k = 31 - __builtin_clz(uint32_t(h + 1));   // heap level of h
            if (nodes[n].cls != -1) {
                // leaf above the bottom: always-right slots lead to this exit
                const int32_t e = ((h + 2) << (depth - k)) - 2 - (S - 1);
                out->exit_class[base + size_t(e)] = -(nodes[n].cls + 1);
                out->exit_leaf[base + size_t(e)] = -(n + 1);
                continue;
            }
            // 1-based heap storage: heap node h lives in slot h + 1 (children 2p, 2p+1)
            out->feature[base + size_t(h) + 1] = nodes[n].feature;
            out->threshold[base + size_t(h) + 1] = nodes[n].threshold;
            for (int32_t b = 0; b < 2; ++b) {
                const int32_t c = nodes[n].left + b;
                const int32_t hc = 2 * h + 1 + b;
                if (hc < (1 << dw) - 1) {
                    slot_node[size_t(hc)] = c;
                } else {
                    // child at the window's last level dw: always-right slots below it
                    // (none when dw = D) lead to its exit
                    const int32_t e = ((hc + 2) << (depth - dw)) - 2 - (S - 1);
                    if (nodes[c].cls != -1) {
                        out->exit_class[base + size_t(e)] = -(nodes[c].cls + 1);
                        out->exit_leaf[base + size_t(e)] = -(c + 1);
                    } else {
                        const int32_t id = int32_t(roots.size());
                        roots.push_back(c);
                        out->exit_class[base + size_t(e)] = id;
                        out->exit_leaf[base + size_t(e)] = id;
                    }
                }
            }
        }
        // A root that is itself a leaf (single-node tree) is handled by the loop above:
        // heap node 0 (slot 1) holds the leaf and its always-right exit is the last one.
    }
}

namespace {

// Exact values of 16-bit float patterns: IEEE binary16 and bfloat16 (the high half of a
// binary32).
double f16_value(uint16_t h) {
    const int e = (h >> 10) & 31;
    const int m = h & 1023;
    const double mag = e == 0    ? std::ldexp(double(m), -24)
                       : e == 31 ? std::numeric_limits<double>::infinity()
                                 : std::ldexp(double(1024 + m), e - 25);
    return (h & 0x8000) ? -mag : mag;
}

double bf16_value(uint16_t h) {
    const uint32_t u = uint32_t(h) << 16;
    float f;
    std::memcpy(&f, &u, 4);
    return double(f);
}

// Smallest non-NaN pattern whose value is >= t (t not NaN).  The non-NaN patterns of a
// sign-magnitude 16-bit format, in increasing value, are indexed 0 .. 2 * inf_bits: index i
// <= inf_bits is the negative magnitude inf_bits - i (-inf up to -0), index i > inf_bits the
// positive magnitude i - inf_bits (the smallest subnormal up to +inf).  Binary search.
template <class Value>
uint16_t round_up_16(float t, int32_t inf_bits, Value value) {
    auto bits = [inf_bits](int32_t i) -> uint16_t {
        return i <= inf_bits ? uint16_t(0x8000 | (inf_bits - i)) : uint16_t(i - inf_bits);
    };
    int32_t lo = 0, hi = 2 * inf_bits;   // +inf is >= every t
    while (lo < hi) {
        const int32_t mid = lo + (hi - lo) / 2;
        if (value(bits(mid)) >= double(t))
            hi = mid;
        else
            lo = mid + 1;
    }
    return bits(lo);
}

}  // namespace

uint32_t narrow_key(float t, dt_dtype type) {
    if (type == DT_U8) {
        if (std::isnan(t) || t <= 0.0f) return 0u;
        if (t > 255.0f) return 256u;
        return uint32_t(std::ceil(t));
    }
    if (type == DT_F16) return std::isnan(t) ? 0x7E00u : round_up_16(t, 0x7C00, f16_value);
    return std::isnan(t) ? 0x7FC0u : round_up_16(t, 0x7F80, bf16_value);
}

void build_narrow_slots(const WindowTables &wt, dt_dtype type, std::vector<uint32_t> *out) {
    const size_t n = wt.threshold.size();
    out->resize(n);
    for (size_t i = 0; i < n; ++i)
        (*out)[i] = (uint32_t(wt.feature[i]) << 16) | narrow_key(wt.threshold[i], type);
}

int64_t data_table_budget(int32_t n_features) {
    int rs = 4;
    while (rs < n_features) rs <<= 1;
    const int64_t tiles = int64_t(2) * 64 * rs * 4;   // two fp32 record tiles of 64 rows
    return std::max<int64_t>(0, std::min<int64_t>(kDataTableBudget, kLdsBytes - tiles));
}

int choose_data_window_depth(const dt_node *nodes, const TreeShape &shape, int64_t max_bytes) {
    // Every window costs a record D steps and an exit lookup, and the records of a
    // wavefront wait for the one with the most windows on its path, so fewer levels are
    // faster as long as the tables stay in the LDS.
    const int max_d = std::min(kMaxWindowDepth, std::max(1, shape.depth));
    int best = 0, smallest = 1;
    int32_t best_levels = 0;
    int64_t best_bytes = 0, smallest_bytes = std::numeric_limits<int64_t>::max();
    for (int d = 1; d <= max_d; ++d) {
        const int64_t bytes = table_bytes(count_windows(nodes, shape, d), d);
        if (bytes <= smallest_bytes) {   // ties: deeper windows
            smallest = d;
            smallest_bytes = bytes;
        }
        if (bytes > max_bytes) continue;
        const int32_t levels = count_levels(nodes, shape, d);
        if (best == 0 || levels < best_levels || (levels == best_levels && bytes < best_bytes)) {
            best = d;
            best_levels = levels;
            best_bytes = bytes;
        }
    }
    return best ? best : smallest;
}

int choose_spec_window_depth(const TreeShape &shape) {
    return std::max(1, std::min(kDefaultSpecWindowDepth, shape.depth));
}

}  // namespace dtree
