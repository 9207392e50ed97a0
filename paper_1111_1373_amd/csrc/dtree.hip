// C ABI of the tree evaluator (include/dtree.h): validation, device upload, launch
// planning and dispatch.  No exception crosses the ABI; errors are status codes plus a
// per-thread message.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "dtree.h"
#include "encode.hpp"
#include "kernels.hpp"
#include "library.hpp"

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

// Device resources of one window encoding: the exits, and the slots once per record
// type (8-byte fp32 slots; 4-byte words on each narrow type's grid).
struct Encoding {
    int32_t depth = 0, n_windows = 0, levels = 0;
    int64_t exit_bytes = 0;                        // padded to 16
    int64_t slot_bytes[dtree::kElemTypes] = {};    // padded to 16
    // [fp32 slots][exit_class][exit_leaf][fp16 slots][bf16 slots][uint8 slots]
    void *d_mem = nullptr;
    const int4 *d_slots[dtree::kElemTypes] = {};
    const int4 *d_exit_class = nullptr;
    const int4 *d_exit_leaf = nullptr;
    int64_t table_bytes(int elem_type) const { return slot_bytes[elem_type] + exit_bytes; }
};

struct DeviceCaps {
    int device = -1;
    int n_cu = 0;
    int lds_per_block = 0;
    int lds_per_cu = 0;
};

dt_status query_device(DeviceCaps *caps) {
    hipError_t e = hipGetDevice(&caps->device);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    e = hipDeviceGetAttribute(&caps->n_cu, hipDeviceAttributeMultiprocessorCount, caps->device);
    if (e != hipSuccess) return hip_fail(e, "hipDeviceGetAttribute(CU count)");
    e = hipDeviceGetAttribute(&caps->lds_per_block, hipDeviceAttributeMaxSharedMemoryPerBlock,
                              caps->device);
    if (e != hipSuccess) return hip_fail(e, "hipDeviceGetAttribute(LDS)");
    e = hipDeviceGetAttribute(&caps->lds_per_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor,
                              caps->device);
    if (e != hipSuccess || caps->lds_per_cu < caps->lds_per_block) caps->lds_per_cu = caps->lds_per_block;
    return DT_OK;
}

dt_status upload_encoding(const dtree::WindowTables &wt, Encoding *enc) {
    enc->depth = wt.depth;
    enc->n_windows = wt.n_windows;
    enc->levels = wt.levels;
    const int64_t n_slots = int64_t(wt.n_windows) * wt.slots;
    enc->exit_bytes = align16(n_slots * 4);
    int64_t off[dtree::kElemTypes];
    int64_t total = 0;
    for (int xt = 0; xt < dtree::kElemTypes; ++xt) {
        enc->slot_bytes[xt] = align16(n_slots * (xt == dtree::kXF32 ? 8 : 4));
        off[xt] = total;
        total += enc->slot_bytes[xt] + (xt == dtree::kXF32 ? 2 * enc->exit_bytes : 0);
    }
    std::vector<unsigned char> host(size_t(total), 0);
    for (int64_t i = 0; i < n_slots; ++i) {
        const int32_t fb = 4 * wt.feature[size_t(i)];   // byte offset in an fp32 row
        std::memcpy(&host[size_t(8 * i)], &wt.threshold[size_t(i)], 4);
        std::memcpy(&host[size_t(8 * i + 4)], &fb, 4);
    }
    const int64_t exit_off = enc->slot_bytes[dtree::kXF32];
    std::memcpy(&host[size_t(exit_off)], wt.exit_class.data(), size_t(n_slots * 4));
    std::memcpy(&host[size_t(exit_off + enc->exit_bytes)], wt.exit_leaf.data(),
                size_t(n_slots * 4));
    std::vector<uint32_t> words;
    for (int xt = dtree::kXF16; xt < dtree::kElemTypes; ++xt) {
        dtree::build_narrow_slots(wt, static_cast<dt_dtype>(xt), &words);
        std::memcpy(&host[size_t(off[xt])], words.data(), size_t(n_slots * 4));
    }
    hipError_t e = hipMalloc(&enc->d_mem, size_t(total));
    if (e != hipSuccess) {
        enc->d_mem = nullptr;
        return fail(DT_ERR_NO_MEMORY, std::string("hipMalloc: ") + hipGetErrorString(e));
    }
    e = hipMemcpy(enc->d_mem, host.data(), size_t(total), hipMemcpyHostToDevice);
    if (e != hipSuccess) return hip_fail(e, "hipMemcpy(tables)");
    auto *base = static_cast<unsigned char *>(enc->d_mem);
    for (int xt = 0; xt < dtree::kElemTypes; ++xt)
        enc->d_slots[xt] = reinterpret_cast<const int4 *>(base + off[xt]);
    enc->d_exit_class = reinterpret_cast<const int4 *>(base + exit_off);
    enc->d_exit_leaf = reinterpret_cast<const int4 *>(base + exit_off + enc->exit_bytes);
    return DT_OK;
}

void free_encoding(Encoding *enc) {
    if (enc->d_mem) (void)hipFree(enc->d_mem);
    enc->d_mem = nullptr;
}

// Pointer-jumping reach per round of the path kernel: entry <- the entry `hops` further
// along.  Procedure 5 reads two further (path[path[path[i]]]).
constexpr int kDefaultPathHops = 2;
constexpr int kMaxPathHops = 8;

dt_status check_options(const dt_tree_options *opt) {
    if (!opt) return DT_OK;
    if (opt->data_window_depth < 0 || opt->data_window_depth > dtree::kMaxWindowDepth)
        return fail(DT_ERR_INVALID_ARG, "data_window_depth must be 0 (auto) or 1..16");
    if (opt->spec_window_depth < 0 || opt->spec_window_depth > dtree::kMaxSpecWindowDepth)
        return fail(DT_ERR_INVALID_ARG, "spec_window_depth must be 0 (auto) or 1..6");
    if (opt->waves_per_cu < 0 || opt->waves_per_cu > 32)
        return fail(DT_ERR_INVALID_ARG, "waves_per_cu must be 0 (auto) or 1..32");
    if (opt->path_hops < 0 || opt->path_hops > kMaxPathHops)
        return fail(DT_ERR_INVALID_ARG, "path_hops must be 0 (auto) or 1..8");
    return DT_OK;
}

void window_depths(const dt_node *nodes, const dtree::TreeShape &shape, int32_t n_features,
                   const dt_tree_options *opt, int *data_d, int *spec_d) {
    *data_d = (opt && opt->data_window_depth)
                  ? opt->data_window_depth
                  : dtree::choose_data_window_depth(nodes, shape,
                                                    dtree::data_table_budget(n_features));
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
    int out_cap = 0;          // single-tree kernels: result tiles buffered per wavefront
    int tile_rows = dtree::kTileRows;   // records per wavefront tile
    int tables_in_lds = 0;
    dt_status status = DT_ERR_UNSUPPORTED;
    std::string why;
};

std::mutex g_prep_mutex;
std::vector<const void *> g_prepared;

// Wavefronts per CU the library aims for (measured on MI355X).  The data decomposition is
// HBM-bound once about 64 KiB of record tiles are in flight per CU; more wavefronts only
// add contention.  The speculative decomposition, which does 2^D times the lane work per
// record, is bound by LDS latency once the tiles are small, and then gains from every
// wavefront up to 16 per CU (uint8 records of 64 features: 207 us with 16 against 282 us
// with 8).  With tiles of 64 fp32 features 64 KiB in flight is again the better point:
// 4 wavefronts of 16 KiB tiles keep a larger result buffer next to the tables (640 us on
// 16,777,216 x 64 records against 674 us with 5), and so do 8 of the 8 KiB tiles of 32
// records that depth-5 and depth-6 windows use (682 us against 726 us with 12 at depth
// 6, 710 against 729 us at depth 5).
// The path reduction is latency-bound and takes as many wavefronts as fit, up to 8.
int target_waves_per_cu(int algo, int tile_bytes) {
    const int hbm = std::max(2, std::min(32, (64 * 1024) / tile_bytes));
    if (algo == DT_ALGO_DATA) return hbm;
    if (algo == DT_ALGO_SPECULATIVE)
        return std::min(16, hbm);
    return 8;
}

void prepare_once(const void *fn, int lds_limit, Plan *plan) {
    std::lock_guard<std::mutex> lock(g_prep_mutex);
    if (std::find(g_prepared.begin(), g_prepared.end(), fn) != g_prepared.end()) return;
    hipError_t e = dtree::prepare_kernel(fn, lds_limit);
    if (e != hipSuccess) {
        plan->why = std::string("hipFuncSetAttribute: ") + hipGetErrorString(e);
        plan->status = DT_ERR_HIP;
        return;
    }
    g_prepared.push_back(fn);
}

// Tables stay in the LDS when that still leaves room for kMinLdsWaves wavefront tiles per
// workgroup; larger trees read their tables from global memory.
constexpr int kMinLdsWaves = 2;
constexpr int kMaxOutCap = 256;

// Single-tree plan: workgroup shape, resident workgroups per CU and the result buffer, for
// records of element type `elem_type` and results of `out_bytes` bytes (1 or 4).  The path
// kernel also keeps its path arrays (kPathIntsPerWave ints per wavefront) after the result
// buffers.
dt_status make_plan(const DeviceCaps &caps, int algo, int elem_type, int row_stride,
                    int load_mode, int depth, int64_t table_bytes, int out_bytes,
                    int waves_per_cu, Plan *plan) {
    const int path_bytes = algo == DT_ALGO_PATH ? dtree::kPathIntsPerWave * 4 : 0;
    const int tile_rows =
        dtree::tile_rows_for(algo, depth, row_stride * dtree::elem_bytes(elem_type));
    plan->tile_rows = tile_rows;
    const int record_tile_bytes = dtree::tile_bytes_for(row_stride, elem_type, tile_rows);
    const int tile_bytes = record_tile_bytes + path_bytes;
    const int res_bytes = tile_rows * out_bytes;   // one tile of results
    if (tile_bytes + res_bytes > caps.lds_per_block) {
        plan->why = "one record tile exceeds the workgroup LDS";
        return plan->status = DT_ERR_UNSUPPORTED;
    }
    const bool tab_lds =
        table_bytes + int64_t(kMinLdsWaves) * (tile_bytes + res_bytes) <= caps.lds_per_block;
    const int table_lds = tab_lds ? int(table_bytes) : 0;
    plan->tables_in_lds = tab_lds ? 1 : 0;
    plan->fn = dtree::kernel_for(algo, elem_type, row_stride, load_mode, tab_lds, depth);
    if (!plan->fn) {
        plan->why = "no kernel instance for this configuration";
        return plan->status = DT_ERR_UNSUPPORTED;
    }
    plan->status = DT_OK;
    prepare_once(plan->fn, caps.lds_per_block, plan);
    if (plan->status != DT_OK) return plan->status;

    const int target =
        waves_per_cu > 0 ? waves_per_cu : target_waves_per_cu(algo, record_tile_bytes);
    // Try every workgroup size and count per CU; keep the shape reaching the most resident
    // wavefronts up to the target (registers and the LDS both limit residency); on ties
    // prefer larger workgroups (fewer table copies), then a larger result buffer.
    int best = 0, best_cap = 0;
    const int max_waves =
        dtree::tree_max_waves(algo, depth, row_stride * dtree::elem_bytes(elem_type));
    for (int w = std::min(max_waves, target); w >= 1; --w) {
        for (int bpc = (target + w - 1) / w; bpc >= 1; --bpc) {
            const int budget = std::min(caps.lds_per_block, caps.lds_per_cu / bpc);
            if (table_lds + w * (tile_bytes + res_bytes) > budget) continue;
            const int cap =
                std::min(kMaxOutCap, (budget - table_lds - w * tile_bytes) / (w * res_bytes));
            const int lds = dtree::lds_bytes_for(table_lds, record_tile_bytes, w, cap * res_bytes) +
                            w * path_bytes;
            int nb = 0;
            hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, plan->fn, w * 64,
                                                                        size_t(lds));
            if (e != hipSuccess) {
                plan->why = std::string("hipOccupancyMaxActiveBlocksPerMultiprocessor: ") +
                            hipGetErrorString(e);
                return plan->status = DT_ERR_HIP;
            }
            const int blocks = std::min(nb, bpc);
            const int score = std::min(target, blocks * w);
            if (blocks >= 1 && (score > best || (score == best && w == plan->waves && cap > best_cap))) {
                best = score;
                best_cap = cap;
                plan->waves = w;
                plan->blocks_per_cu = blocks;
                plan->lds_bytes = lds;
                plan->out_cap = cap;
            }
        }
    }
    if (best == 0) {
        plan->why = "tables and one record tile exceed the workgroup LDS";
        return plan->status = DT_ERR_UNSUPPORTED;
    }
    plan->why.clear();
    return plan->status = DT_OK;
}

}  // namespace

struct dt_tree {
    DeviceCaps caps;
    dtree::TreeShape shape;
    int32_t n_features = 0, n_classes = 0;
    int row_stride = 0;
    int path_hops = kDefaultPathHops;
    Encoding enc[2];              // data windows, speculative windows (also the path kernel's)
    // [algo][record element type][load mode][uint8 / int32 results]
    Plan plan[3][dtree::kElemTypes][dtree::kLoadModes][2];
};

// Encoding an algorithm runs on: the path kernel reduces the speculative windows.
static inline int encoding_of(int algo) { return algo == DT_ALGO_DATA ? 0 : 1; }

static bool single_tree_algo(dt_algo algo) {
    return algo == DT_ALGO_DATA || algo == DT_ALGO_SPECULATIVE || algo == DT_ALGO_PATH;
}

namespace {

// Device resources of a forest for one decomposition: all trees' window tables back to
// back (tree k: slots then class exits, each padded to 16 bytes), the per-tree
// descriptors {byte_off, slot_bytes, levels, 0} and the LDS chunks
// {first_tree, end_tree, byte_off, bytes}.
struct ForestEncoding {
    int32_t depth = 0;
    void *d_mem = nullptr;
    const int4 *d_tables = nullptr, *d_trees = nullptr, *d_chunks = nullptr;
    const int2 *d_roots = nullptr;
    std::vector<int4> trees;     // host copy of the descriptors
    std::vector<int2> roots;     // per tree: slot 1 of window 0 {threshold bits, feature bytes}
    std::vector<int4> chunks;    // host copy of the chunks
    int64_t table_bytes = 0;
    int64_t max_tree_bytes = 0;
    int32_t chunk_lds_bytes = 0; // LDS reserved for one chunk (0: tables read in place)
    int32_t waves = 0;           // wavefronts per workgroup (one tile each)
    int exit_mode = 0;           // exit codes: int32 table (0), int16 table (1), or packed
                                 // into the windows' bottom slots (2)
};

void free_forest_encoding(ForestEncoding *e) {
    if (e->d_mem) (void)hipFree(e->d_mem);
    e->d_mem = nullptr;
}

}  // namespace

struct dt_forest {
    DeviceCaps caps;
    int32_t n_trees = 0, n_features = 0, n_classes = 0;
    int row_stride = 0;
    int vote_words = 0;
    ForestEncoding enc[2];       // [DT_ALGO_DATA], [DT_ALGO_SPECULATIVE]
    Plan plan[2][dtree::kLoadModes];  // [algo][load mode]
};

namespace {

// The fastest record-tile load path the layout of the features allows.
int load_mode_for(const void *d_x, int elem_type, int64_t ld, int32_t n_features,
                  int row_stride) {
    const bool dense = ld == n_features && (n_features * dtree::elem_bytes(elem_type)) % 16 == 0 &&
                       (reinterpret_cast<uintptr_t>(d_x) & 15u) == 0;
    if (!dense) return dtree::kLoadScalar;
    return n_features == row_stride ? dtree::kLoadExact : dtree::kLoadVec;
}

uint32_t magic_div(int32_t d) {
    return d >= 2 ? uint32_t(((uint64_t(1) << 32) + uint64_t(d) - 1) / uint64_t(d)) : 0u;
}

dtree::Rows make_rows(const void *d_x, int elem_type, int64_t n, int64_t ld, int32_t n_features,
                      int tile_rows = dtree::kTileRows) {
    dtree::Rows r{};
    r.x = d_x;
    r.n = n;
    r.ld = ld;
    r.n_tiles = (n + tile_rows - 1) / tile_rows;
    r.n_features = n_features;
    r.magic_f = magic_div(n_features);
    r.n_words = n_features * dtree::elem_bytes(elem_type) / 4;   // used by vector loads only
    r.magic_w = magic_div(r.n_words);
    return r;
}

bool valid_elem_type(dt_dtype t) {
    return t == DT_F32 || t == DT_F16 || t == DT_BF16 || t == DT_U8;
}

dt_status classify_impl(const dt_tree *tree, const void *d_x, dt_dtype x_type, int64_t n,
                        int64_t ld, void *d_out, dt_output out_kind, dt_algo algo, void *stream) {
    if (!tree) return fail(DT_ERR_INVALID_ARG, "tree is NULL");
    if (n < 0) return fail(DT_ERR_INVALID_ARG, "n must be >= 0");
    if (!single_tree_algo(algo)) return fail(DT_ERR_INVALID_ARG, "unknown algo");
    if (!valid_elem_type(x_type)) return fail(DT_ERR_INVALID_ARG, "unknown x_type");
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

    if ((reinterpret_cast<uintptr_t>(d_x) % uintptr_t(dtree::elem_bytes(x_type))) != 0)
        return fail(DT_ERR_INVALID_ARG, "d_x is not aligned to its element size");
    const int mode = load_mode_for(d_x, x_type, ld, tree->n_features, tree->row_stride);
    const Plan &plan = tree->plan[algo][x_type][mode][out_kind == DT_OUT_CLASS_U8 ? 0 : 1];
    if (plan.status != DT_OK) return fail(plan.status, plan.why);
    const Encoding &enc = tree->enc[encoding_of(algo)];

    dtree::KArgs a{};
    a.in = make_rows(d_x, x_type, n, ld, tree->n_features, plan.tile_rows);
    a.slots = enc.d_slots[x_type];
    a.exits = out_kind == DT_OUT_LEAF_I32 ? enc.d_exit_leaf : enc.d_exit_class;
    a.slot_bytes = int32_t(enc.slot_bytes[x_type]);
    a.exit_bytes = int32_t(enc.exit_bytes);
    a.depth = enc.depth;
    a.levels = enc.levels;
    a.waves = plan.waves;
    a.out_kind = out_kind == DT_OUT_CLASS_U8 ? 0 : 1;
    a.out_cap = plan.out_cap;
    a.out_vec = (reinterpret_cast<uintptr_t>(d_out) & 15u) == 0 ? 1 : 0;
    a.hops = tree->path_hops;
    a.out = d_out;
    const int64_t want = (a.in.n_tiles + plan.waves - 1) / plan.waves;
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
    if (opt && opt->path_hops) t->path_hops = opt->path_hops;
    int depth[2];
    window_depths(nodes, shape, n_features, opt, &depth[0], &depth[1]);
    for (int e = 0; e < 2; ++e) {
        dtree::WindowTables wt;
        dtree::build_windows(nodes, shape, depth[e], &wt);
        st = upload_encoding(wt, &t->enc[e]);
        if (st != DT_OK) {
            free_encoding(&t->enc[0]);
            free_encoding(&t->enc[1]);
            delete t;
            return st;
        }
    }
    for (int algo = 0; algo < 3; ++algo) {
        const Encoding &enc = t->enc[encoding_of(algo)];
        for (int xt = 0; xt < dtree::kElemTypes; ++xt) {
            for (int m = 0; m < dtree::kLoadModes; ++m) {
                Plan *pl = t->plan[algo][xt][m];
                if (t->row_stride > dtree::kMaxRowStride) {
                    pl[0].why = pl[1].why = "n_features > 256";
                    continue;
                }
                if (algo == DT_ALGO_PATH && xt != DT_F32) {
                    pl[0].why = pl[1].why = "the path kernel reads fp32 records only";
                    continue;
                }
                if (m == dtree::kLoadExact && n_features != t->row_stride) continue;
                if (m != dtree::kLoadScalar && (n_features * dtree::elem_bytes(xt)) % 16 != 0)
                    continue;
                for (int o = 0; o < 2; ++o)
                    make_plan(t->caps, algo, xt, t->row_stride, m, enc.depth, enc.table_bytes(xt),
                              o == 0 ? 1 : 4, opt ? opt->waves_per_cu : 0, &pl[o]);
            }
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

// ---- forests ---------------------------------------------------------------------------

// Speculative forests use windows of depth 2 (default) or 4.
constexpr int kForestSpecDepth = 2;

int vote_words_for(int32_t n_classes) {
    if (n_classes <= 8) return 2;
    if (n_classes <= 16) return 4;
    return 16;
}

// Encode every tree with window depth `depth` and lay the tables out back to back.
void encode_forest(const dt_node *nodes, const int32_t *offsets, int32_t n_trees,
                   const std::vector<dtree::TreeShape> &shapes, int algo, int depth,
                   std::vector<unsigned char> *bytes, ForestEncoding *enc) {
    enc->depth = depth;
    enc->trees.assign(size_t(n_trees), int4{0, 0, 0, 0});
    enc->roots.assign(size_t(n_trees), int2{0, 0});
    enc->max_tree_bytes = 0;
    bytes->clear();
    std::vector<dtree::WindowTables> wts(static_cast<size_t>(n_trees));
    // Exit codes (next window ids, and results -(class + 1)) of the data decomposition are
    // packed into the spare bits of the windows' bottom slots when every code of the forest
    // fits 11 bits (the feature's byte offset, at most 1020, takes the low 10): the tables
    // then hold slots only, a fifth less than with int16 codes (four complete depth-10
    // trees per 32 KiB chunk instead of three), and the walk reads no exit table.  Failing
    // that they are int16 when every code fits, else int32.  (The speculative walk keeps
    // int32 codes: its narrower instances need more registers than 16 wavefronts per CU
    // leave it.)
    bool fits11 = algo == DT_ALGO_DATA, fits16 = algo == DT_ALGO_DATA;
    for (int32_t k = 0; k < n_trees; ++k) {
        dtree::build_windows(nodes + offsets[k], shapes[size_t(k)], depth, &wts[size_t(k)]);
        for (int32_t c : wts[size_t(k)].exit_class) {
            fits11 = fits11 && c >= -1024 && c <= 1023;
            fits16 = fits16 && c >= INT16_MIN && c <= INT16_MAX;
        }
    }
    enc->exit_mode = fits11 ? 2 : fits16 ? 1 : 0;
    const int64_t exit_size = enc->exit_mode == 2 ? 0 : enc->exit_mode == 1 ? 2 : 4;
    for (int32_t k = 0; k < n_trees; ++k) {
        const dtree::WindowTables &wt = wts[size_t(k)];
        const int64_t n_slots = int64_t(wt.n_windows) * wt.slots;
        const int64_t sb = align16(n_slots * 8), eb = align16(n_slots * exit_size);
        const int64_t off = int64_t(bytes->size());
        bytes->resize(size_t(off + sb + eb), 0);
        unsigned char *p = bytes->data() + off;
        const int64_t S = wt.slots;
        for (int64_t i = 0; i < n_slots; ++i) {
            int32_t fb = 4 * wt.feature[size_t(i)];   // byte offset in an fp32 row
            const int64_t q = i % S;                  // heap position in the window
            if (enc->exit_mode == 2 && q >= S / 2) {  // bottom level: its children's exits
                const int64_t e = i - q + 2 * q - S;  // exit of child 2q in this window
                const uint32_t lo = uint32_t(wt.exit_class[size_t(e)]) & 0x7FFu;
                const uint32_t hi = uint32_t(wt.exit_class[size_t(e + 1)]) & 0x7FFu;
                fb = int32_t(uint32_t(fb) | lo << 10 | hi << 21);
            }
            std::memcpy(p + 8 * i, &wt.threshold[size_t(i)], 4);
            std::memcpy(p + 8 * i + 4, &fb, 4);
        }
        if (enc->exit_mode == 1) {
            for (int64_t i = 0; i < n_slots; ++i) {
                const int16_t c = int16_t(wt.exit_class[size_t(i)]);
                std::memcpy(p + sb + 2 * i, &c, 2);
            }
        } else if (enc->exit_mode == 0) {
            std::memcpy(p + sb, wt.exit_class.data(), size_t(n_slots * 4));
        }
        enc->trees[size_t(k)] = int4{int(off), int(sb), wt.levels, 0};
        int2 root{0, 0};                          // the slot just written for slot 1
        std::memcpy(&root, p + 8, 8);
        enc->roots[size_t(k)] = root;
        enc->max_tree_bytes = std::max(enc->max_tree_bytes, sb + eb);
    }
    enc->table_bytes = int64_t(bytes->size());
}

// Wavefronts per CU the forest kernel aims for by default (measured: 16 beat 8 by 5% on a
// 32-tree forest; more gained nothing).
constexpr int kForestWavesPerCu = 16;

// Choose the workgroup shape and the LDS chunks of consecutive trees.
void chunk_forest(const DeviceCaps &caps, int algo, int row_stride, int waves_per_cu,
                  ForestEncoding *enc) {
    const int64_t tile_bytes = dtree::tile_bytes_for(row_stride, dtree::kXF32);
    const int target = waves_per_cu > 0 ? waves_per_cu : kForestWavesPerCu;
    enc->chunks.clear();
    // Workgroup shape: the most resident wavefronts up to the target whose tiles leave a
    // chunk buffer that holds the largest tree; ties: larger chunk buffers (fewer passes).
    int best_w = 0, best_score = 0;
    int64_t best_budget = 0;
    for (int bpc = 1; bpc <= 4; ++bpc) {
        const int64_t per_block = std::min<int64_t>(caps.lds_per_block, caps.lds_per_cu / bpc);
        for (int w = dtree::forest_max_waves(algo, enc->depth, row_stride); w >= 1; --w) {
            const int64_t budget = per_block - w * tile_bytes;
            if (budget < enc->max_tree_bytes) continue;
            const int score = std::min(target, w * bpc);
            if (score > best_score || (score == best_score && budget > best_budget)) {
                best_w = w;
                best_score = score;
                best_budget = budget;
            }
        }
    }
    if (best_w > 0) {
        const int w = best_w;
        const int64_t budget = best_budget;
        enc->waves = w;
        int32_t first = 0;
        int64_t max_chunk = 0;
        while (first < int32_t(enc->trees.size())) {
            int32_t end = first;
            int64_t bytes = 0;
            while (end < int32_t(enc->trees.size())) {
                const int64_t off = enc->trees[size_t(end)].x;
                const int64_t next = end + 1 < int32_t(enc->trees.size())
                                         ? int64_t(enc->trees[size_t(end + 1)].x)
                                         : enc->table_bytes;
                if (bytes + (next - off) > budget) break;
                bytes += next - off;
                ++end;
            }
            const int32_t off0 = enc->trees[size_t(first)].x;
            enc->chunks.push_back(int4{first, end, off0, int(bytes)});
            max_chunk = std::max(max_chunk, bytes);
            first = end;
        }
        enc->chunk_lds_bytes = int32_t(max_chunk);
        return;
    }
    // single trees too large for the LDS: one pass reading the tables in place
    enc->waves = 0;
    enc->chunk_lds_bytes = 0;
    enc->chunks.push_back(int4{0, int(enc->trees.size()), 0, int(enc->table_bytes)});
}

dt_status upload_forest(const std::vector<unsigned char> &bytes, ForestEncoding *enc) {
    const int64_t tb = align16(int64_t(bytes.size()));
    const int64_t db = int64_t(enc->trees.size()) * 16;
    const int64_t cb = int64_t(enc->chunks.size()) * 16;
    const int64_t rb = int64_t(enc->roots.size()) * 8;
    std::vector<unsigned char> host(size_t(tb + db + cb + rb), 0);
    std::memcpy(host.data(), bytes.data(), bytes.size());
    std::memcpy(host.data() + tb, enc->trees.data(), size_t(db));
    std::memcpy(host.data() + tb + db, enc->chunks.data(), size_t(cb));
    std::memcpy(host.data() + tb + db + cb, enc->roots.data(), size_t(rb));
    hipError_t e = hipMalloc(&enc->d_mem, host.size());
    if (e != hipSuccess) {
        enc->d_mem = nullptr;
        return fail(DT_ERR_NO_MEMORY, std::string("hipMalloc: ") + hipGetErrorString(e));
    }
    e = hipMemcpy(enc->d_mem, host.data(), host.size(), hipMemcpyHostToDevice);
    if (e != hipSuccess) return hip_fail(e, "hipMemcpy(forest tables)");
    auto *base = static_cast<unsigned char *>(enc->d_mem);
    enc->d_tables = reinterpret_cast<const int4 *>(base);
    enc->d_trees = reinterpret_cast<const int4 *>(base + tb);
    enc->d_chunks = reinterpret_cast<const int4 *>(base + tb + db);
    enc->d_roots = reinterpret_cast<const int2 *>(base + tb + db + cb);
    return DT_OK;
}

dt_status plan_forest(const DeviceCaps &caps, int algo, int row_stride, int load_mode,
                      int vote_words, const ForestEncoding &enc, Plan *plan) {
    const bool tab_lds = enc.chunk_lds_bytes > 0;
    plan->fn = dtree::forest_kernel_for(algo, row_stride, load_mode, tab_lds, vote_words,
                                        enc.depth, enc.exit_mode);
    if (!plan->fn) {
        plan->why = "no forest kernel instance for this configuration";
        return plan->status = DT_ERR_UNSUPPORTED;
    }
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
    for (int w = 1; w <= dtree::forest_max_waves(algo, enc.depth, row_stride); ++w) {
        if (tab_lds && w != enc.waves) continue;     // the chunks were cut for enc.waves
        const int lds = dtree::lds_bytes_for(enc.chunk_lds_bytes,
                                             dtree::tile_bytes_for(row_stride, dtree::kXF32), w);
        if (lds > caps.lds_per_block) break;
        int nb = 0;
        hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, plan->fn, w * 64,
                                                                    size_t(lds));
        if (e != hipSuccess) {
            plan->why = std::string("hipOccupancyMaxActiveBlocksPerMultiprocessor: ") +
                        hipGetErrorString(e);
            return plan->status = DT_ERR_HIP;
        }
        if (nb >= 1 && nb * w >= best_waves) {
            best_waves = nb * w;
            plan->waves = w;
            plan->blocks_per_cu = nb;
            plan->lds_bytes = lds;
        }
    }
    if (best_waves == 0) {
        plan->why = "no workgroup shape fits this forest kernel";
        return plan->status = DT_ERR_UNSUPPORTED;
    }
    plan->why.clear();
    return plan->status = DT_OK;
}

void forest_destroy_impl(dt_forest *f) {
    if (!f) return;
    free_forest_encoding(&f->enc[0]);
    free_forest_encoding(&f->enc[1]);
    delete f;
}

dt_status forest_create_impl(const dt_node *nodes, const int32_t *offsets, int32_t n_trees,
                             int32_t n_features, int32_t n_classes, const dt_tree_options *opt,
                             dt_forest **out) {
    if (!out) return fail(DT_ERR_INVALID_ARG, "out is NULL");
    if (!nodes || !offsets) return fail(DT_ERR_INVALID_ARG, "nodes or tree_offsets is NULL");
    if (n_trees < 1) return fail(DT_ERR_INVALID_ARG, "n_trees must be >= 1");
    if (n_features < 1 || n_classes < 1)
        return fail(DT_ERR_INVALID_ARG, "n_features and n_classes must be >= 1");
    dt_status st = check_options(opt);
    if (st != DT_OK) return st;
    if (opt && opt->spec_window_depth != 0 && opt->spec_window_depth != 2 &&
        opt->spec_window_depth != 4)
        return fail(DT_ERR_UNSUPPORTED, "forests use speculative windows of depth 2 or 4");
    if (n_trees > dtree::kMaxForestTrees)
        return fail(DT_ERR_UNSUPPORTED, "forests are limited to 255 trees");
    if (n_classes > dtree::kMaxForestClasses)
        return fail(DT_ERR_UNSUPPORTED, "forests are limited to 64 classes");
    if (offsets[0] != 0) return fail(DT_ERR_INVALID_ARG, "tree_offsets[0] must be 0");
    std::vector<dtree::TreeShape> shapes(static_cast<size_t>(n_trees));
    int max_depth = 0;
    for (int32_t k = 0; k < n_trees; ++k) {
        if (offsets[k + 1] <= offsets[k])
            return fail(DT_ERR_INVALID_ARG, "tree_offsets must increase strictly");
        std::string msg;
        st = dtree::validate_tree(nodes + offsets[k], offsets[k + 1] - offsets[k], n_features,
                                  n_classes, &shapes[size_t(k)], &msg);
        if (st != DT_OK) return fail(st, "tree " + std::to_string(k) + ": " + msg);
        max_depth = std::max(max_depth, shapes[size_t(k)].depth);
    }
    dt_forest *f = new (std::nothrow) dt_forest();
    if (!f) return fail(DT_ERR_NO_MEMORY, "host allocation failed");
    st = query_device(&f->caps);
    if (st != DT_OK) { delete f; return st; }
    f->n_trees = n_trees;
    f->n_features = n_features;
    f->n_classes = n_classes;
    f->row_stride = row_stride_for(n_features);
    f->vote_words = vote_words_for(n_classes);

    // data windows: the depth that makes the forest's tables smallest
    int data_d = opt && opt->data_window_depth ? opt->data_window_depth : 0;
    if (!data_d) {
        int64_t best = -1;
        for (int d = 1; d <= std::min(dtree::kMaxWindowDepth, std::max(1, max_depth)); ++d) {
            int64_t total = 0;
            for (int32_t k = 0; k < n_trees; ++k)
                total += dtree::table_bytes(
                    dtree::count_windows(nodes + offsets[k], shapes[size_t(k)], d), d);
            if (best < 0 || total <= best) { best = total; data_d = d; }
        }
    }
    const int spec_d = opt && opt->spec_window_depth ? opt->spec_window_depth : kForestSpecDepth;
    const int depth[2] = {data_d, spec_d};
    for (int algo = 0; algo < 2; ++algo) {
        std::vector<unsigned char> bytes;
        encode_forest(nodes, offsets, n_trees, shapes, algo, depth[algo], &bytes, &f->enc[algo]);
        if (f->row_stride <= dtree::kMaxRowStride)
            chunk_forest(f->caps, algo, f->row_stride, opt ? opt->waves_per_cu : 0,
                         &f->enc[algo]);
        else
            f->enc[algo].chunks.push_back(int4{0, n_trees, 0, int(f->enc[algo].table_bytes)});
        if (f->enc[algo].table_bytes > (int64_t(1) << 31) - 1) {
            forest_destroy_impl(f);
            return fail(DT_ERR_UNSUPPORTED, "forest tables exceed 2 GiB");
        }
        st = upload_forest(bytes, &f->enc[algo]);
        if (st != DT_OK) { forest_destroy_impl(f); return st; }
        for (int m = 0; m < dtree::kLoadModes; ++m) {
            if (f->row_stride > dtree::kMaxRowStride) {
                f->plan[algo][m].why = "n_features > 256";
                continue;
            }
            if (m == dtree::kLoadExact && n_features != f->row_stride) continue;
            if (m != dtree::kLoadScalar && n_features % 4 != 0) continue;
            plan_forest(f->caps, algo, f->row_stride, m, f->vote_words, f->enc[algo],
                        &f->plan[algo][m]);
        }
    }
    *out = f;
    return DT_OK;
}

dt_status forest_classify_impl(const dt_forest *f, const float *d_x, int64_t n, int64_t ld,
                               void *d_out, dt_output out_kind, dt_algo algo, void *stream) {
    if (!f) return fail(DT_ERR_INVALID_ARG, "forest is NULL");
    if (n < 0) return fail(DT_ERR_INVALID_ARG, "n must be >= 0");
    if (algo == DT_ALGO_PATH)
        return fail(DT_ERR_UNSUPPORTED, "forests run the data and speculative decompositions");
    if (algo != DT_ALGO_DATA && algo != DT_ALGO_SPECULATIVE)
        return fail(DT_ERR_INVALID_ARG, "unknown algo");
    if (out_kind != DT_OUT_CLASS_U8 && out_kind != DT_OUT_CLASS_I32)
        return fail(DT_ERR_INVALID_ARG, "forests output classes (uint8 or int32)");
    if (ld < f->n_features) return fail(DT_ERR_INVALID_ARG, "ld must be >= n_features");
    if (f->n_features > dtree::kMaxRowStride)
        return fail(DT_ERR_UNSUPPORTED, "n_features > 256");
    if (n > (int64_t(1) << 37)) return fail(DT_ERR_UNSUPPORTED, "n > 2^37");
    if (n == 0) return DT_OK;
    if (!d_x || !d_out) return fail(DT_ERR_INVALID_ARG, "null device pointer");
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev != f->caps.device)
        return fail(DT_ERR_INVALID_ARG, "current device differs from the forest's device");
    const Plan &plan =
        f->plan[algo][load_mode_for(d_x, dtree::kXF32, ld, f->n_features, f->row_stride)];
    if (plan.status != DT_OK) return fail(plan.status, plan.why);
    const ForestEncoding &enc = f->enc[algo];

    dtree::FArgs a{};
    a.in = make_rows(d_x, dtree::kXF32, n, ld, f->n_features);
    a.tables = enc.d_tables;
    a.trees = enc.d_trees;
    a.roots = enc.d_roots;
    a.chunks = enc.d_chunks;
    a.n_trees = f->n_trees;
    a.n_chunks = int32_t(enc.chunks.size());
    a.table_lds_bytes = enc.chunk_lds_bytes;
    a.depth = enc.depth;
    a.n_classes = f->n_classes;
    a.waves = plan.waves;
    a.out_kind = out_kind == DT_OUT_CLASS_U8 ? 0 : 1;
    a.out = d_out;
    const int64_t groups = (a.in.n_tiles + plan.waves - 1) / plan.waves;
    const int64_t resident = int64_t(plan.blocks_per_cu) * f->caps.n_cu;
    const int blocks = int(std::max<int64_t>(1, std::min(groups, resident)));
    e = dtree::launch_forest(plan.fn, a, blocks, plan.lds_bytes, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "forest kernel launch");
    return DT_OK;
}

}  // namespace

namespace dtree {

dt_status set_error(dt_status s, const std::string &msg) { return fail(s, msg); }
dt_status set_hip_error(hipError_t e, const char *what) { return hip_fail(e, what); }
void clear_error() { g_last_error.clear(); }
int device_of(const dt_tree *t) { return t->caps.device; }
int device_of(const dt_forest *f) { return f->caps.device; }
int32_t features_of(const dt_tree *t) { return t->n_features; }
int32_t features_of(const dt_forest *f) { return f->n_features; }

}  // namespace dtree

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
            window_depths(nodes, shape, n_features, opt, &dd, &sd);
            fill_info(shape, n_features, n_classes, dd, dtree::count_windows(nodes, shape, dd),
                      dtree::count_levels(nodes, shape, dd), sd, dtree::count_windows(nodes, shape, sd),
                      dtree::count_levels(nodes, shape, sd), info);
        }
        return DT_OK;
    } catch (const std::bad_alloc &) {
        return fail(DT_ERR_NO_MEMORY, "host allocation failed");
    } catch (...) {
        return fail(DT_ERR_INVALID_ARG, "unexpected internal error");
    }
}

dt_status dt_threshold_keys(const float *thresholds, int64_t n, dt_dtype type, uint16_t *keys) {
    g_last_error.clear();
    if (n < 0) return fail(DT_ERR_INVALID_ARG, "n must be >= 0");
    if (type != DT_F16 && type != DT_BF16 && type != DT_U8)
        return fail(DT_ERR_INVALID_ARG, "type must be DT_F16, DT_BF16 or DT_U8");
    if (n > 0 && (!thresholds || !keys)) return fail(DT_ERR_INVALID_ARG, "null buffer");
    for (int64_t i = 0; i < n; ++i) keys[i] = uint16_t(dtree::narrow_key(thresholds[i], type));
    return DT_OK;
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
        if (levels) *levels = dtree::count_levels(nodes, shape, window_depth);
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

dt_status dt_tree_launch_info(const dt_tree *t, const void *d_x, dt_dtype x_type, int64_t ld,
                              dt_output out_kind, dt_algo algo, dt_launch_info *info) {
    g_last_error.clear();
    if (!t || !info) return fail(DT_ERR_INVALID_ARG, "null argument");
    if (!single_tree_algo(algo)) return fail(DT_ERR_INVALID_ARG, "unknown algo");
    if (!valid_elem_type(x_type)) return fail(DT_ERR_INVALID_ARG, "unknown x_type");
    if (out_kind != DT_OUT_CLASS_U8 && out_kind != DT_OUT_CLASS_I32 && out_kind != DT_OUT_LEAF_I32)
        return fail(DT_ERR_INVALID_ARG, "unknown out_kind");
    if (ld < t->n_features) return fail(DT_ERR_INVALID_ARG, "ld must be >= n_features");
    const int mode = load_mode_for(d_x, x_type, ld, t->n_features, t->row_stride);
    const Plan &plan = t->plan[algo][x_type][mode][out_kind == DT_OUT_CLASS_U8 ? 0 : 1];
    if (plan.status != DT_OK) return fail(plan.status, plan.why);
    info->waves_per_workgroup = plan.waves;
    info->workgroups_per_cu = plan.blocks_per_cu;
    info->lds_bytes = plan.lds_bytes;
    info->result_buffer_tiles = plan.out_cap;
    info->tables_in_lds = plan.tables_in_lds;
    info->load_mode = mode;
    info->tile_rows = plan.tile_rows;
    return DT_OK;
}

dt_status dt_classify(const dt_tree *t, const float *d_x, int64_t n, int64_t ld, void *d_out,
                      dt_output out_kind, dt_algo algo, void *stream) {
    try {
        g_last_error.clear();
        return classify_impl(t, d_x, DT_F32, n, ld, d_out, out_kind, algo, stream);
    } catch (...) {
        return fail(DT_ERR_INVALID_ARG, "unexpected internal error");
    }
}

dt_status dt_classify_typed(const dt_tree *t, const void *d_x, dt_dtype x_type, int64_t n,
                            int64_t ld, void *d_out, dt_output out_kind, dt_algo algo,
                            void *stream) {
    try {
        g_last_error.clear();
        return classify_impl(t, d_x, x_type, n, ld, d_out, out_kind, algo, stream);
    } catch (...) {
        return fail(DT_ERR_INVALID_ARG, "unexpected internal error");
    }
}

dt_status dt_forest_create(const dt_node *nodes, const int32_t *tree_offsets, int32_t n_trees,
                           int32_t n_features, int32_t n_classes, const dt_tree_options *opt,
                           dt_forest **out) {
    try {
        g_last_error.clear();
        return forest_create_impl(nodes, tree_offsets, n_trees, n_features, n_classes, opt, out);
    } catch (const std::bad_alloc &) {
        return fail(DT_ERR_NO_MEMORY, "host allocation failed");
    } catch (...) {
        return fail(DT_ERR_INVALID_ARG, "unexpected internal error");
    }
}

void dt_forest_destroy(dt_forest *f) { forest_destroy_impl(f); }

dt_status dt_forest_classify(const dt_forest *f, const float *d_x, int64_t n, int64_t ld,
                             void *d_out, dt_output out_kind, dt_algo algo, void *stream) {
    try {
        g_last_error.clear();
        return forest_classify_impl(f, d_x, n, ld, d_out, out_kind, algo, stream);
    } catch (...) {
        return fail(DT_ERR_INVALID_ARG, "unexpected internal error");
    }
}

}  // extern "C"
