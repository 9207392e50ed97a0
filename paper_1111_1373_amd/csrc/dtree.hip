// C ABI of the tree evaluator (include/dtree.h): validation, device upload, launch
// planning and dispatch.  No exception crosses the ABI; errors are status codes plus a
// per-thread message.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "dtree.h"
#include "encode.hpp"
#include "kernels.hpp"

namespace {

thread_local std::string g_last_error;

dt_status fail(dt_status s, const std::string &msg) {
    g_last_error = msg;
    return s;
}

dt_status hip_fail(hipError_t e, const char *what) {
    return fail(DT_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

inline int64_t align16(int64_t b) { return (b + 15) & ~int64_t(15); }

int row_stride_for(int32_t n_features) {
    int rs = 4;
    while (rs < n_features) rs <<= 1;
    return rs;
}

// Device resources of one window encoding.
struct Encoding {
    int32_t depth = 0, n_windows = 0, levels = 0;
    int64_t slot_bytes = 0, exit_bytes = 0;   // padded to 16
    void *d_mem = nullptr;                    // [slots][exit_class][exit_leaf]
    const int4 *d_slots = nullptr;
    const int4 *d_exit_class = nullptr;
    const int4 *d_exit_leaf = nullptr;
    int64_t table_bytes() const { return slot_bytes + exit_bytes; }
};

struct DeviceCaps {
    int device = -1;
    int n_cu = 0;
    int lds_per_block = 0;
};

dt_status query_device(DeviceCaps *caps) {
    hipError_t e = hipGetDevice(&caps->device);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    e = hipDeviceGetAttribute(&caps->n_cu, hipDeviceAttributeMultiprocessorCount, caps->device);
    if (e != hipSuccess) return hip_fail(e, "hipDeviceGetAttribute(CU count)");
    e = hipDeviceGetAttribute(&caps->lds_per_block, hipDeviceAttributeMaxSharedMemoryPerBlock,
                              caps->device);
    if (e != hipSuccess) return hip_fail(e, "hipDeviceGetAttribute(LDS)");
    return DT_OK;
}

dt_status upload_encoding(const dtree::WindowTables &wt, Encoding *enc) {
    enc->depth = wt.depth;
    enc->n_windows = wt.n_windows;
    enc->levels = wt.levels;
    const int64_t n_slots = int64_t(wt.n_windows) * wt.slots;
    enc->slot_bytes = align16(n_slots * 8);
    enc->exit_bytes = align16(n_slots * 4);
    const int64_t total = enc->slot_bytes + 2 * enc->exit_bytes;
    std::vector<unsigned char> host(size_t(total), 0);
    for (int64_t i = 0; i < n_slots; ++i) {
        std::memcpy(&host[size_t(8 * i)], &wt.threshold[size_t(i)], 4);
        std::memcpy(&host[size_t(8 * i + 4)], &wt.feature[size_t(i)], 4);
    }
    std::memcpy(&host[size_t(enc->slot_bytes)], wt.exit_class.data(), size_t(n_slots * 4));
    std::memcpy(&host[size_t(enc->slot_bytes + enc->exit_bytes)], wt.exit_leaf.data(),
                size_t(n_slots * 4));
    hipError_t e = hipMalloc(&enc->d_mem, size_t(total));
    if (e != hipSuccess) {
        enc->d_mem = nullptr;
        return fail(DT_ERR_NO_MEMORY, std::string("hipMalloc: ") + hipGetErrorString(e));
    }
    e = hipMemcpy(enc->d_mem, host.data(), size_t(total), hipMemcpyHostToDevice);
    if (e != hipSuccess) return hip_fail(e, "hipMemcpy(tables)");
    auto *base = static_cast<unsigned char *>(enc->d_mem);
    enc->d_slots = reinterpret_cast<const int4 *>(base);
    enc->d_exit_class = reinterpret_cast<const int4 *>(base + enc->slot_bytes);
    enc->d_exit_leaf = reinterpret_cast<const int4 *>(base + enc->slot_bytes + enc->exit_bytes);
    return DT_OK;
}

void free_encoding(Encoding *enc) {
    if (enc->d_mem) (void)hipFree(enc->d_mem);
    enc->d_mem = nullptr;
}

dt_status check_options(const dt_tree_options *opt) {
    if (!opt) return DT_OK;
    if (opt->data_window_depth < 0 || opt->data_window_depth > dtree::kMaxWindowDepth)
        return fail(DT_ERR_INVALID_ARG, "data_window_depth must be 0 (auto) or 1..16");
    if (opt->spec_window_depth < 0 || opt->spec_window_depth > dtree::kMaxSpecWindowDepth)
        return fail(DT_ERR_INVALID_ARG, "spec_window_depth must be 0 (auto) or 1..6");
    return DT_OK;
}

void window_depths(const dt_node *nodes, const dtree::TreeShape &shape,
                   const dt_tree_options *opt, int *data_d, int *spec_d) {
    *data_d = (opt && opt->data_window_depth) ? opt->data_window_depth
                                              : dtree::choose_data_window_depth(nodes, shape);
    *spec_d = (opt && opt->spec_window_depth) ? opt->spec_window_depth
                                              : dtree::choose_spec_window_depth(shape);
}

void fill_info(const dtree::TreeShape &shape, int32_t n_features, int32_t n_classes,
               int data_d, int64_t data_w, int32_t data_lv, int spec_d, int64_t spec_w,
               int32_t spec_lv, dt_tree_info *info) {
    info->n_nodes = shape.n_nodes;
    info->n_internal = shape.n_internal;
    info->n_leaves = shape.n_leaves;
    info->depth = shape.depth;
    info->n_features = n_features;
    info->n_classes = n_classes;
    info->data_window_depth = data_d;
    info->data_windows = int32_t(data_w);
    info->data_levels = data_lv;
    info->spec_window_depth = spec_d;
    info->spec_windows = int32_t(spec_w);
    info->spec_levels = spec_lv;
    info->data_table_bytes = align16(data_w * (int64_t(1) << data_d) * 8) +
                             align16(data_w * (int64_t(1) << data_d) * 4);
    info->spec_table_bytes = align16(spec_w * (int64_t(1) << spec_d) * 8) +
                             align16(spec_w * (int64_t(1) << spec_d) * 4);
}

// Launch plan of one kernel instance: wavefronts per workgroup and resident workgroups.
struct Plan {
    const void *fn = nullptr;
    int waves = 0;
    int blocks_per_cu = 0;
    int lds_bytes = 0;
    dt_status status = DT_ERR_UNSUPPORTED;
    std::string why;
};

std::mutex g_prep_mutex;
std::vector<const void *> g_prepared;

// Plan for one kernel instance with the tables either in the LDS or in global memory.
dt_status plan_variant(const DeviceCaps &caps, int algo, int row_stride, bool vec, int depth,
                       bool tab_lds, int64_t table_bytes, Plan *plan) {
    plan->fn = dtree::kernel_for(algo, row_stride, vec, tab_lds, depth);
    if (!plan->fn) {
        plan->why = "no kernel instance for this configuration";
        return plan->status = DT_ERR_UNSUPPORTED;
    }
    const int lds_tables = tab_lds ? int(table_bytes) : 0;
    {
        std::lock_guard<std::mutex> lock(g_prep_mutex);
        if (std::find(g_prepared.begin(), g_prepared.end(), plan->fn) == g_prepared.end()) {
            hipError_t e = dtree::prepare_kernel(plan->fn, caps.lds_per_block);
            if (e != hipSuccess) {
                plan->why = std::string("hipFuncSetAttribute: ") + hipGetErrorString(e);
                return plan->status = DT_ERR_HIP;
            }
            g_prepared.push_back(plan->fn);
        }
    }
    int best_waves = 0;
    for (int w = 1; w <= dtree::kMaxWavesPerBlock; ++w) {
        const int lds = dtree::lds_bytes_for(lds_tables, row_stride, w);
        if (lds > caps.lds_per_block) break;
        int nb = 0;
        hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, plan->fn, w * 64,
                                                                    size_t(lds));
        if (e != hipSuccess) {
            plan->why = std::string("hipOccupancyMaxActiveBlocksPerMultiprocessor: ") +
                        hipGetErrorString(e);
            return plan->status = DT_ERR_HIP;
        }
        if (nb < 1) continue;
        if (nb * w >= best_waves) {   // ties: larger workgroups share one table copy
            best_waves = nb * w;
            plan->waves = w;
            plan->blocks_per_cu = nb;
            plan->lds_bytes = lds;
        }
    }
    if (best_waves == 0) {
        plan->why = "no workgroup shape fits this kernel";
        return plan->status = DT_ERR_UNSUPPORTED;
    }
    plan->why.clear();
    return plan->status = DT_OK;
}

// Tables stay in the LDS when that still leaves room for kMinLdsWaves wavefront tiles per
// workgroup; larger trees read their tables from global memory.
constexpr int kMinLdsWaves = 2;

dt_status make_plan(const DeviceCaps &caps, int algo, int row_stride, bool vec, int depth,
                    int64_t table_bytes, Plan *plan) {
    if (dtree::lds_bytes_for(0, row_stride, 1) > caps.lds_per_block) {
        plan->why = "one record tile exceeds the workgroup LDS";
        return plan->status = DT_ERR_UNSUPPORTED;
    }
    const bool fits = table_bytes + int64_t(kMinLdsWaves) * dtree::kTileRows * row_stride * 4 <=
                      caps.lds_per_block;
    return plan_variant(caps, algo, row_stride, vec, depth, fits, table_bytes, plan);
}

}  // namespace

struct dt_tree {
    DeviceCaps caps;
    dtree::TreeShape shape;
    int32_t n_features = 0, n_classes = 0;
    int row_stride = 0;
    Encoding enc[2];              // [DT_ALGO_DATA], [DT_ALGO_SPECULATIVE]
    Plan plan[2][2];              // [algo][vectorised]
};

struct dt_forest {
    int32_t n_trees = 0;
    std::vector<dt_tree *> trees;
};

namespace {

dt_status classify_impl(const dt_tree *tree, const float *d_x, int64_t n, int64_t ld,
                        void *d_out, dt_output out_kind, dt_algo algo, void *stream) {
    if (!tree) return fail(DT_ERR_INVALID_ARG, "tree is NULL");
    if (n < 0) return fail(DT_ERR_INVALID_ARG, "n must be >= 0");
    if (algo != DT_ALGO_DATA && algo != DT_ALGO_SPECULATIVE)
        return fail(DT_ERR_INVALID_ARG, "unknown algo");
    if (out_kind != DT_OUT_CLASS_U8 && out_kind != DT_OUT_CLASS_I32 &&
        out_kind != DT_OUT_LEAF_I32)
        return fail(DT_ERR_INVALID_ARG, "unknown out_kind");
    if (ld < tree->n_features) return fail(DT_ERR_INVALID_ARG, "ld must be >= n_features");
    if (out_kind == DT_OUT_CLASS_U8 && tree->n_classes > 256)
        return fail(DT_ERR_INVALID_ARG, "uint8 output needs n_classes <= 256");
    if (tree->n_features > dtree::kMaxRowStride)
        return fail(DT_ERR_UNSUPPORTED, "n_features > 256");
    if (n > (int64_t(1) << 37)) return fail(DT_ERR_UNSUPPORTED, "n > 2^37");
    if (n == 0) return DT_OK;
    if (!d_x || !d_out) return fail(DT_ERR_INVALID_ARG, "null device pointer");
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev != tree->caps.device)
        return fail(DT_ERR_INVALID_ARG, "current device differs from the tree's device");

    const bool vec = (ld == tree->n_features) && (tree->n_features % 4 == 0) &&
                     ((reinterpret_cast<uintptr_t>(d_x) & 15u) == 0);
    const Plan &plan = tree->plan[algo][vec ? 1 : 0];
    if (plan.status != DT_OK) return fail(plan.status, plan.why);
    const Encoding &enc = tree->enc[algo];

    dtree::KArgs a{};
    a.x = d_x;
    a.n = n;
    a.ld = ld;
    a.n_tiles = (n + dtree::kTileRows - 1) / dtree::kTileRows;
    a.n_features = tree->n_features;
    a.magic_f = tree->n_features >= 2
                    ? uint32_t(((uint64_t(1) << 32) + uint64_t(tree->n_features) - 1) /
                               uint64_t(tree->n_features))
                    : 0u;
    a.slots = enc.d_slots;
    a.exits = out_kind == DT_OUT_LEAF_I32 ? enc.d_exit_leaf : enc.d_exit_class;
    a.slot_bytes = int32_t(enc.slot_bytes);
    a.exit_bytes = int32_t(enc.exit_bytes);
    a.depth = enc.depth;
    a.levels = enc.levels;
    a.waves = plan.waves;
    a.out_kind = out_kind == DT_OUT_CLASS_U8 ? 0 : 1;
    a.out = d_out;
    const int64_t want = (a.n_tiles + plan.waves - 1) / plan.waves;
    const int64_t resident = int64_t(plan.blocks_per_cu) * tree->caps.n_cu;
    const int blocks = int(std::max<int64_t>(1, std::min(want, resident)));
    e = dtree::launch_kernel(plan.fn, a, blocks, plan.lds_bytes,
                             static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "kernel launch");
    return DT_OK;
}

dt_status create_impl(const dt_node *nodes, int32_t n_nodes, int32_t n_features,
                      int32_t n_classes, const dt_tree_options *opt, dt_tree **out) {
    if (!out) return fail(DT_ERR_INVALID_ARG, "out is NULL");
    dt_status st = check_options(opt);
    if (st != DT_OK) return st;
    std::string msg;
    dtree::TreeShape shape;
    st = dtree::validate_tree(nodes, n_nodes, n_features, n_classes, &shape, &msg);
    if (st != DT_OK) return fail(st, msg);
    dt_tree *t = new (std::nothrow) dt_tree();
    if (!t) return fail(DT_ERR_NO_MEMORY, "host allocation failed");
    st = query_device(&t->caps);
    if (st != DT_OK) { delete t; return st; }
    t->shape = shape;
    t->n_features = n_features;
    t->n_classes = n_classes;
    t->row_stride = row_stride_for(n_features);
    int depth[2];
    window_depths(nodes, shape, opt, &depth[0], &depth[1]);
    for (int algo = 0; algo < 2; ++algo) {
        dtree::WindowTables wt;
        dtree::build_windows(nodes, shape, depth[algo], &wt);
        st = upload_encoding(wt, &t->enc[algo]);
        if (st != DT_OK) {
            free_encoding(&t->enc[0]);
            free_encoding(&t->enc[1]);
            delete t;
            return st;
        }
        for (int v = 0; v < 2; ++v) {
            if (t->row_stride > dtree::kMaxRowStride) {
                t->plan[algo][v].why = "n_features > 256";
                continue;
            }
            make_plan(t->caps, algo, t->row_stride, v == 1, t->enc[algo].depth,
                      t->enc[algo].table_bytes(), &t->plan[algo][v]);
        }
    }
    *out = t;
    return DT_OK;
}

void destroy_impl(dt_tree *t) {
    if (!t) return;
    free_encoding(&t->enc[0]);
    free_encoding(&t->enc[1]);
    delete t;
}

}  // namespace

extern "C" {

int32_t dt_abi_version(void) { return DT_ABI_VERSION; }

const char *dt_status_string(dt_status s) {
    switch (s) {
        case DT_OK: return "ok";
        case DT_ERR_INVALID_ARG: return "invalid argument";
        case DT_ERR_INVALID_TREE: return "invalid tree";
        case DT_ERR_UNSUPPORTED: return "unsupported";
        case DT_ERR_HIP: return "HIP runtime error";
        case DT_ERR_NO_MEMORY: return "out of memory";
        default: return "unknown status";
    }
}

const char *dt_last_error(void) { return g_last_error.c_str(); }

dt_status dt_tree_check(const dt_node *nodes, int32_t n_nodes, int32_t n_features,
                        int32_t n_classes, const dt_tree_options *opt, dt_tree_info *info) {
    try {
        g_last_error.clear();
        dt_status st = check_options(opt);
        if (st != DT_OK) return st;
        std::string msg;
        dtree::TreeShape shape;
        st = dtree::validate_tree(nodes, n_nodes, n_features, n_classes, &shape, &msg);
        if (st != DT_OK) return fail(st, msg);
        if (info) {
            int dd, sd;
            window_depths(nodes, shape, opt, &dd, &sd);
            fill_info(shape, n_features, n_classes, dd, dtree::count_windows(nodes, shape, dd),
                      dtree::count_levels(shape, dd), sd, dtree::count_windows(nodes, shape, sd),
                      dtree::count_levels(shape, sd), info);
        }
        return DT_OK;
    } catch (const std::bad_alloc &) {
        return fail(DT_ERR_NO_MEMORY, "host allocation failed");
    } catch (...) {
        return fail(DT_ERR_INVALID_ARG, "unexpected internal error");
    }
}

dt_status dt_encode_windows(const dt_node *nodes, int32_t n_nodes, int32_t n_features,
                            int32_t n_classes, int32_t window_depth, int32_t capacity_windows,
                            int32_t *features, float *thresholds, int32_t *exit_class,
                            int32_t *exit_leaf, int32_t *n_windows, int32_t *levels) {
    try {
        g_last_error.clear();
        if (window_depth < 1 || window_depth > dtree::kMaxWindowDepth)
            return fail(DT_ERR_INVALID_ARG, "window_depth must be 1..16");
        if (capacity_windows < 0) return fail(DT_ERR_INVALID_ARG, "capacity_windows < 0");
        std::string msg;
        dtree::TreeShape shape;
        dt_status st = dtree::validate_tree(nodes, n_nodes, n_features, n_classes, &shape, &msg);
        if (st != DT_OK) return fail(st, msg);
        const int64_t nw = dtree::count_windows(nodes, shape, window_depth);
        if (nw * (int64_t(1) << window_depth) > (int64_t(1) << 30))
            return fail(DT_ERR_UNSUPPORTED, "window tables too large");
        if (n_windows) *n_windows = int32_t(nw);
        if (levels) *levels = dtree::count_levels(shape, window_depth);
        if (capacity_windows == 0) return DT_OK;
        if (capacity_windows < nw) return fail(DT_ERR_INVALID_ARG, "capacity_windows too small");
        if (!features || !thresholds || !exit_class || !exit_leaf)
            return fail(DT_ERR_INVALID_ARG, "null output buffer");
        dtree::WindowTables wt;
        dtree::build_windows(nodes, shape, window_depth, &wt);
        const size_t ns = wt.feature.size();
        std::memcpy(features, wt.feature.data(), ns * 4);
        std::memcpy(thresholds, wt.threshold.data(), ns * 4);
        std::memcpy(exit_class, wt.exit_class.data(), ns * 4);
        std::memcpy(exit_leaf, wt.exit_leaf.data(), ns * 4);
        return DT_OK;
    } catch (const std::bad_alloc &) {
        return fail(DT_ERR_NO_MEMORY, "host allocation failed");
    } catch (...) {
        return fail(DT_ERR_INVALID_ARG, "unexpected internal error");
    }
}

dt_status dt_tree_create(const dt_node *nodes, int32_t n_nodes, int32_t n_features,
                         int32_t n_classes, const dt_tree_options *opt, dt_tree **out) {
    try {
        g_last_error.clear();
        return create_impl(nodes, n_nodes, n_features, n_classes, opt, out);
    } catch (const std::bad_alloc &) {
        return fail(DT_ERR_NO_MEMORY, "host allocation failed");
    } catch (...) {
        return fail(DT_ERR_INVALID_ARG, "unexpected internal error");
    }
}

dt_status dt_tree_get_info(const dt_tree *t, dt_tree_info *info) {
    g_last_error.clear();
    if (!t || !info) return fail(DT_ERR_INVALID_ARG, "null argument");
    fill_info(t->shape, t->n_features, t->n_classes, t->enc[0].depth, t->enc[0].n_windows,
              t->enc[0].levels, t->enc[1].depth, t->enc[1].n_windows, t->enc[1].levels, info);
    return DT_OK;
}

void dt_tree_destroy(dt_tree *t) { destroy_impl(t); }

dt_status dt_classify(const dt_tree *t, const float *d_x, int64_t n, int64_t ld, void *d_out,
                      dt_output out_kind, dt_algo algo, void *stream) {
    try {
        g_last_error.clear();
        return classify_impl(t, d_x, n, ld, d_out, out_kind, algo, stream);
    } catch (...) {
        return fail(DT_ERR_INVALID_ARG, "unexpected internal error");
    }
}

dt_status dt_forest_create(const dt_node *nodes, const int32_t *tree_offsets, int32_t n_trees,
                           int32_t n_features, int32_t n_classes, const dt_tree_options *opt,
                           dt_forest **out) {
    g_last_error.clear();
    (void)nodes; (void)tree_offsets; (void)n_trees; (void)n_features; (void)n_classes;
    (void)opt; (void)out;
    return fail(DT_ERR_UNSUPPORTED, "forests are not implemented yet");
}

void dt_forest_destroy(dt_forest *f) {
    if (!f) return;
    for (dt_tree *t : f->trees) destroy_impl(t);
    delete f;
}

dt_status dt_forest_classify(const dt_forest *f, const float *d_x, int64_t n, int64_t ld,
                             void *d_out, dt_output out_kind, dt_algo algo, void *stream) {
    g_last_error.clear();
    (void)f; (void)d_x; (void)n; (void)ld; (void)d_out; (void)out_kind; (void)algo; (void)stream;
    return fail(DT_ERR_UNSUPPORTED, "forests are not implemented yet");
}

}  // extern "C"
