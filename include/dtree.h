/*
 * dtree.h -- C ABI of the MI355X (gfx950) classification-tree evaluator.
 *
 * Evaluates a trained full binary classification tree with continuous-attribute tests
 * over every record of an fp32 feature matrix, following Spencer, "Speculative Parallel
 * Evaluation of Classification Trees on GPGPU Compute Engines":
 *   - DT_ALGO_DATA: the data decomposition of Section 3.2 (Procedure 3): one GPU lane
 *     per record walks the tree without branches.
 *   - DT_ALGO_SPECULATIVE: the speculative decomposition of Sections 3.3-3.4
 *     (Procedures 4-5): a group of lanes evaluates every decision node of a block of
 *     the tree for one record at once, the per-node outcomes are gathered into a
 *     64-bit wavefront mask, and the reached node is found by walking the mask.  Trees
 *     deeper than one block are evaluated block after block (the "window" of
 *     Section 6).
 *   - DT_ALGO_PATH: the same speculative evaluation, reduced as Procedure 5 prints it:
 *     a path array in the LDS, leaves pointing to themselves, pointer jumping until the
 *     root's entry names a leaf.  Kept to compare the paper's mechanism with the mask.
 *   - Forests (Section 1, trees evaluated one after another and combined): majority
 *     vote, ties to the smallest class id.
 *
 * Decision rule: a record x goes to the LEFT child of node n iff x[feature_n] <
 * threshold_n, and to the RIGHT child otherwise.  Ties (x == t) and NaN features go
 * right.  IEEE comparison: -0.0 == +0.0, denormals are not flushed.  The paper states
 * the complementary form (left iff x <= t); a tree in that form converts exactly by
 * replacing each threshold t by nextafterf(t, +inf) (for t < +inf).
 *
 * Tree layout: the breadth-first array of Procedure 1 (Section 3.1).  Node i stores
 * its feature, threshold, the index of its LEFT child and a class; the right child is
 * left + 1.  A decision node has cls == -1 (the paper's "no class").  Procedure 1 emits
 * exactly this layout; any node order is accepted as long as every child index is
 * larger than its parent's index, every node but the root has exactly one parent, and
 * the tree is full (every decision node has two children).
 *
 * Threading: handles are immutable after creation; classify calls on the same handle
 * may run concurrently on different streams.  All calls are noexcept: no C++ exception
 * crosses the ABI.  The last error message of the calling thread is available from
 * dt_last_error().
 */
#ifndef DTREE_H
#define DTREE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DT_ABI_VERSION 6

typedef enum {
    DT_OK = 0,
    DT_ERR_INVALID_ARG = 1,   /* null pointer, negative size, ld < n_features, bad enum   */
    DT_ERR_INVALID_TREE = 2,  /* not a full binary tree in the layout above, or a feature
                                 or class out of range                                     */
    DT_ERR_UNSUPPORTED = 3,   /* valid input beyond this library's limits (see below)     */
    DT_ERR_HIP = 4,           /* a HIP runtime call failed                                 */
    DT_ERR_NO_MEMORY = 5      /* host or device allocation failed                          */
} dt_status;

typedef enum {
    DT_ALGO_DATA = 0,         /* one lane per record (Procedure 3)                          */
    DT_ALGO_SPECULATIVE = 1,  /* lanes per decision node, predicate mask walk (Proc. 4-5)  */
    DT_ALGO_PATH = 2          /* lanes per decision node, path array reduced by pointer
                                 jumping as printed in Procedure 5 (single trees only)      */
} dt_algo;

typedef enum {
    DT_OUT_CLASS_U8 = 0,      /* uint8_t label per record; requires n_classes <= 256      */
    DT_OUT_CLASS_I32 = 1,     /* int32_t label per record                                   */
    DT_OUT_LEAF_I32 = 2       /* int32_t index (in the node array) of the leaf reached;
                                 single trees only                                          */
} dt_output;

/*
 * Element type of the records (dt_classify_typed).  Section 2.1 treats continuous
 * attributes as real values carried in floating point and notes that ordered discrete
 * values behave the same; narrower record types cut the bytes read per record.  Every
 * element is widened exactly to fp32 and compared with the fp32 threshold, so the result
 * is the fp32 result for the widened records.
 */
typedef enum {
    DT_F32 = 0,               /* IEEE binary32                                              */
    DT_F16 = 1,               /* IEEE binary16 (bits in a uint16)                           */
    DT_BF16 = 2,              /* bfloat16: the upper 16 bits of a binary32                  */
    DT_U8 = 3                 /* uint8: ordered discrete values 0..255                      */
} dt_dtype;

/* One node of the breadth-first array (Procedure 1).  16 bytes, no padding. */
typedef struct {
    int32_t feature;    /* 0-based attribute index (the paper counts from 1); decision nodes */
    float threshold;    /* any float, including +-inf and NaN; decision nodes               */
    int32_t left;       /* index of the left child; right child = left + 1; decision nodes  */
    int32_t cls;        /* class in [0, n_classes) for a leaf, -1 for a decision node        */
} dt_node;

typedef struct dt_tree dt_tree;
typedef struct dt_forest dt_forest;

/*
 * Evaluation layout options.  Both decompositions cut the tree into blocks ("windows",
 * Section 6) of at most `depth` levels, each embedded in a complete subtree of 2^depth - 1
 * slots.  0 selects the library's choice.
 *   data_window_depth: 1..16.  Default: the fewest window levels whose tables take at
 *     most 48 KiB (and leave the LDS room for two fp32 record tiles); ties go to smaller
 *     tables; if no depth fits, the depth with the smallest tables.
 *   spec_window_depth: 1..6 (a window has at most 63 decision nodes, one 64-lane
 *     wavefront).  2^depth lanes evaluate one record, so 64 / 2^depth records share a
 *     wavefront instruction.  Default: 2 (4 lanes per record, measured fastest), or the
 *     tree depth if smaller; 4 gives the paper's record groups of 16 lanes (15 decision
 *     nodes and one idle lane, Section 4.2).  Forests accept 2 (default) or 4.
 */
typedef struct {
    int32_t data_window_depth;
    int32_t spec_window_depth;
    int32_t waves_per_cu;      /* launch tuning: resident wavefronts per compute unit
                                  (0 = the library's choice, about 64 KiB of record tiles in
                                  flight per CU); limited by the LDS and registers */
    int32_t path_hops;         /* DT_ALGO_PATH: entries read further along per reduction
                                  round, 1..8 (0 = 2: path[i] <- path[path[path[i]]], the
                                  form printed in Procedure 5) */
} dt_tree_options;

/* Shape of a tree and of its two encodings. */
typedef struct {
    int32_t n_nodes, n_internal, n_leaves;
    int32_t depth;                  /* edges on the longest root-to-leaf path            */
    int32_t n_features, n_classes;
    int32_t data_window_depth, data_windows, data_levels;
    int32_t spec_window_depth, spec_windows, spec_levels;
    int64_t data_table_bytes, spec_table_bytes;   /* bytes staged in LDS per workgroup  */
} dt_tree_info;

/* Version of this ABI (DT_ABI_VERSION of the header the library was built from). */
int32_t dt_abi_version(void);

/* Static description of a status code.  Never NULL. */
const char *dt_status_string(dt_status s);

/* Detailed message of the calling thread's last failed call ("" if none).  The pointer
 * stays valid until the thread's next dt_* call. */
const char *dt_last_error(void);

/*
 * Validate a tree and describe its encodings.  Host only: touches no GPU.
 *   nodes      host array of n_nodes records (read only; not retained)
 *   opt        may be NULL (defaults)
 *   info       out, may be NULL
 * Errors: DT_ERR_INVALID_ARG (null nodes, n_nodes < 1, n_features < 1, n_classes < 1,
 * option out of range), DT_ERR_INVALID_TREE (see the layout rules above),
 * DT_ERR_UNSUPPORTED (n_nodes > 2^24).
 */
dt_status dt_tree_check(const dt_node *nodes, int32_t n_nodes, int32_t n_features,
                        int32_t n_classes, const dt_tree_options *opt, dt_tree_info *info);

/*
 * Window encoding used by the GPU kernels, written to caller-owned host buffers.  Host
 * only.  Window w occupies slots [w*2^d, (w+1)*2^d) of each array (d = window_depth):
 *   features[], thresholds[]  slot p in [1, 2^d) is node p of the window's heap, stored
 *                   1-based: the window root is slot 1 and the children of slot p are
 *                   slots 2p and 2p+1.  A slot that holds no decision node has feature 0
 *                   and threshold -inf, so it always sends a record right.  Slot 0 is
 *                   padding with the same values.
 *   exit_class[], exit_leaf[]  entry e is the outcome of leaving the window at bottom
 *                   position e (heap position 2^d + e): a value v >= 0 is the window
 *                   to continue in; v < 0 ends the walk with class (resp. leaf index)
 *                   -v - 1.  A leaf met above the bottom level is recorded at the exit
 *                   reached by always going right from it.
 * Window 0 is rooted at node 0; windows are numbered in breadth-first order of their roots.
 * Windows are rooted at tree depth 0 and at depths d0, d0 + d, d0 + 2d, ...: window 0 holds
 * d0 <= d levels (its slots below them always go right), every other window d.  d0 is d,
 * unless the shallower d0 = depth - d * (levels - 1), which fills the deepest level of
 * windows instead of the first, needs fewer windows (Section 6 leaves the cut points open).
 * Call with capacity_windows = 0 (buffers may be NULL) to learn *n_windows and *levels
 * (the largest number of windows on a root-to-leaf path).  Errors as dt_tree_check, plus
 * DT_ERR_INVALID_ARG for window_depth outside 1..16 or a capacity below *n_windows with
 * non-zero capacity.
 */
dt_status dt_encode_windows(const dt_node *nodes, int32_t n_nodes, int32_t n_features,
                            int32_t n_classes, int32_t window_depth, int32_t capacity_windows,
                            int32_t *features, float *thresholds, int32_t *exit_class,
                            int32_t *exit_leaf, int32_t *n_windows, int32_t *levels);

/*
 * Keys the kernels for narrow records compare against (host only).  Records of type fp16,
 * bf16 or uint8 are compared in their own type: each threshold t is moved onto the type's
 * grid, rounded up, as key[i]:
 *   DT_F16, DT_BF16  the bits of the smallest non-NaN value of the type that is >= t
 *                    (-0 for t = 0; +inf above the largest finite value); a NaN threshold
 *                    gives a quiet NaN (0x7E00, 0x7FC0).
 *   DT_U8            the smallest integer k in 0..256 with k >= t; 0 for t <= 0 or NaN.
 * No value of the type lies in [t, key), so for every record value x the kernels'
 * test "x < key" (fp16/bf16) or "x < key" on integers (uint8) equals the decision x < t of
 * Procedure 1 on the widened value, and a NaN t sends every record right either way.
 *   thresholds  host array of n floats; keys: host array of n uint16 (caller-owned)
 * Errors: DT_ERR_INVALID_ARG for n < 0, null buffers with n > 0, or a type other than
 * DT_F16, DT_BF16, DT_U8.
 */
dt_status dt_threshold_keys(const float *thresholds, int64_t n, dt_dtype type, uint16_t *keys);

/*
 * Upload a tree (Section 3.1: the breadth-first node array of Procedure 1, evaluated by
 * the recursive descent of Section 2.1; Section 3.3: the decision nodes the speculative
 * decomposition maps to lanes).  Validate it, encode it for both decompositions and copy
 * the encodings to the current HIP device.  Synchronous: the upload is complete on
 * return.  The caller keeps ownership of `nodes`.  The handle owns its device memory and
 * is bound to the device that was current at creation.
 * Errors: as dt_tree_check, DT_ERR_HIP, DT_ERR_NO_MEMORY.  *out is set only on DT_OK.
 */
dt_status dt_tree_create(const dt_node *nodes, int32_t n_nodes, int32_t n_features,
                         int32_t n_classes, const dt_tree_options *opt, dt_tree **out);

/* Describe a created tree.  Errors: DT_ERR_INVALID_ARG (null). */
dt_status dt_tree_get_info(const dt_tree *tree, dt_tree_info *info);

/* Free a tree and its device memory.  NULL is a no-op.  No classify call on the tree may
 * still be in flight (synchronise its streams first). */
void dt_tree_destroy(dt_tree *tree);

/* Launch shape dt_classify uses for one (algorithm, output, input layout).  Diagnostic. */
typedef struct {
    int32_t waves_per_workgroup;
    int32_t workgroups_per_cu;     /* resident workgroups per compute unit               */
    int32_t lds_bytes;             /* dynamic LDS per workgroup                          */
    int32_t result_buffer_tiles;   /* tiles of results each wavefront buffers           */
    int32_t tables_in_lds;         /* 1: tree tables staged in the LDS, 0: read in place */
    int32_t load_mode;             /* 0: scalar loads, 1: 16-byte loads, 2: 16-byte loads
                                      of rows exactly one LDS row stride wide            */
    int32_t tile_rows;             /* records per wavefront tile: 64, or 32 for the
                                      speculative walk of 64-slot windows on rows of at
                                      least 32 bytes                                     */
} dt_launch_info;

/* Fill *info with the launch shape of dt_classify_typed(tree, d_x, x_type, n, ld, ...,
 * out_kind, algo) for any n > 0.  Only the alignment of d_x is read.  Errors:
 * DT_ERR_INVALID_ARG (null, unknown enum, ld < n_features), or the error classify would
 * return for this shape. */
dt_status dt_tree_launch_info(const dt_tree *tree, const void *d_x, dt_dtype x_type,
                              int64_t ld, dt_output out_kind, dt_algo algo,
                              dt_launch_info *info);

/*
 * Classify n records: the label of the leaf each record reaches from the root, taking the
 * left child when x[feature] < threshold (Section 2.1's evaluation; Section 3.2,
 * Procedure 3 for DT_ALGO_DATA; Sections 3.3-3.4, Procedures 4-5 for DT_ALGO_SPECULATIVE
 * and DT_ALGO_PATH).  Asynchronous on `stream` (a hipStream_t; NULL = the null stream).
 *   d_x     device pointer, row-major fp32, record r at d_x + r*ld, columns
 *           0..n_features-1 are read.  Any alignment of 4 bytes; rows that are
 *           contiguous (ld == n_features), a multiple of 4 floats and 16-byte aligned
 *           take the vectorised load path.
 *   n       number of records, >= 0 (0: nothing is launched)
 *   ld      row stride in floats, >= n_features
 *   d_out   device pointer to n labels of the type named by out_kind
 *   algo    DT_ALGO_DATA, DT_ALGO_SPECULATIVE or DT_ALGO_PATH; all give identical
 *           results
 * Exactly n outputs are written; nothing is written on an error return.  Buffers are
 * owned by the caller and must stay valid until the work on `stream` completes.  The call
 * puts one kernel launch on `stream` and nothing else (no allocation, copy, memset or
 * synchronisation), so it may be captured in a HIP graph; a tree handle is never written
 * after creation, so calls on several streams may use it at once.
 * Errors: DT_ERR_INVALID_ARG (null tree or pointers with n > 0, n < 0, ld < n_features,
 * unknown enum, DT_OUT_CLASS_U8 with n_classes > 256, device other than the tree's),
 * DT_ERR_UNSUPPORTED (n_features > 256, n > 2^37), DT_ERR_HIP (launch failure).
 * A tree's tables are staged in the LDS when they fit next to the record tiles and are
 * read from global memory otherwise; every valid tree is supported.
 */
dt_status dt_classify(const dt_tree *tree, const float *d_x, int64_t n, int64_t ld,
                      void *d_out, dt_output out_kind, dt_algo algo, void *stream);

/*
 * dt_classify for narrow records (Section 2.1: ordered discrete attributes behave like the
 * real-valued ones).  Records of element type x_type (dt_dtype): d_x must be aligned to the
 * element size and ld counts elements.  Rows that are contiguous, 16-byte aligned and a
 * multiple of 16 bytes long take the vectorised load path.  Each element is widened
 * exactly to fp32 before its comparison, so the labels equal those of dt_classify on the
 * widened records.  DT_ALGO_PATH reads DT_F32 records only (DT_ERR_UNSUPPORTED otherwise).
 * Errors: as dt_classify, and DT_ERR_INVALID_ARG for an unknown x_type or a misaligned d_x.
 */
dt_status dt_classify_typed(const dt_tree *tree, const void *d_x, dt_dtype x_type, int64_t n,
                            int64_t ld, void *d_out, dt_output out_kind, dt_algo algo,
                            void *stream);

/*
 * Upload a forest: several trees evaluated one after another and combined (Section 1,
 * the concatenated-trees scheme it cites), each tree in the layout of Procedure 1
 * (Section 3.1).  Tree k occupies nodes[tree_offsets[k] .. tree_offsets[k+1])
 * with child indices local to that range (each tree is a valid array on its own).
 * tree_offsets has n_trees + 1 entries, starts at 0 and increases strictly.  All trees
 * share n_features and n_classes.  Synchronous upload, as dt_tree_create.
 * Errors: as dt_tree_create; DT_ERR_INVALID_ARG for bad offsets or n_trees < 1;
 * DT_ERR_UNSUPPORTED for n_trees > 255 or n_classes > 64.
 */
dt_status dt_forest_create(const dt_node *nodes, const int32_t *tree_offsets,
                           int32_t n_trees, int32_t n_features, int32_t n_classes,
                           const dt_tree_options *opt, dt_forest **out);

/* Free a forest.  NULL is a no-op.  Same in-flight rule as dt_tree_destroy. */
void dt_forest_destroy(dt_forest *forest);

/*
 * Majority vote of the forest's trees for n records; ties go to the smallest class id
 * (Section 1's forests; each tree evaluated as dt_classify, Sections 3.2-3.4).
 * Arguments, errors, graph capture and concurrent use as dt_classify; out_kind must be
 * DT_OUT_CLASS_U8 or DT_OUT_CLASS_I32.
 */
dt_status dt_forest_classify(const dt_forest *forest, const float *d_x, int64_t n, int64_t ld,
                             void *d_out, dt_output out_kind, dt_algo algo, void *stream);

/* ---- host-resident records: the outer-time path -------------------------------------
 *
 * Section 4.2 times each GPU function twice: the "outer" time of the whole call (device
 * allocation, host-to-device copy of the records, kernel, copy of the labels back, free)
 * and the "inner" time of the kernel alone; Section 4.3 finds the serial copies dominate
 * and names pinned host buffers and copies overlapped with computation as the remedy.
 * A dt_pipeline does that for records that live in host memory: it owns n_slots device
 * chunk buffers (and pinned bounce buffers), and for each chunk of chunk_rows records it
 * copies the rows in, classifies them and copies the labels out on the slot's own
 * stream, so the copies of one chunk overlap the kernel and the copies of the others.
 * With `serial` set it instead does what Section 4.2 describes: allocate device buffers
 * for all n records, copy in, classify, copy out and free, one step after the other.
 */
typedef struct dt_pipeline dt_pipeline;

typedef struct {
    int64_t chunk_rows;   /* records per chunk (0: about 32 MiB of features; rounded up
                             to a multiple of 64) */
    int32_t n_slots;      /* chunks in flight, 1..8 (0 = 3) */
    int32_t serial;       /* 1: per-call allocation and serial copies, as Section 4.2;
                             chunk_rows, n_slots and host_threads are then unused */
    int32_t host_threads; /* host threads that copy pageable records into the pinned
                             buffers, 1..16 (0 = 4) */
} dt_pipeline_options;

/* Timing of a call, host wall clock and HIP events (microseconds).  Chunks overlap, so
 * the per-step sums can exceed outer_us. */
typedef struct {
    double outer_us;      /* wall clock of the whole call, copies included              */
    double kernel_us;     /* sum over chunks of the classify kernel's duration          */
    double h2d_us;        /* sum over chunks of the record copy's duration              */
    double d2h_us;        /* sum over chunks of the label copy's duration               */
    int64_t chunks;
    int32_t input_pinned; /* 1: the records were copied straight from the caller's
                             buffer (page-locked); 0: through pinned bounce buffers     */
    int32_t output_pinned;
} dt_pipeline_stats;

/*
 * Pipeline for records of n_features floats, on the current device (Section 4.3's remedy
 * for copy-dominated outer time: pinned host buffers and copies overlapped with the
 * kernels).  Allocates its device
 * and pinned host buffers and creates its streams (default priority) here, never in a
 * call (unless `serial`).  opt may be NULL.
 * Errors: DT_ERR_INVALID_ARG (null out, n_features not 1..256, option out of range),
 * DT_ERR_NO_MEMORY, DT_ERR_HIP.
 */
dt_status dt_pipeline_create(int32_t n_features, const dt_pipeline_options *opt,
                             dt_pipeline **out);

/* Free a pipeline (Section 4.3's overlapped copies; waits for its streams first).  NULL is
 * a no-op. */
void dt_pipeline_destroy(dt_pipeline *pipeline);

/*
 * Outer-time classification (Section 4.2: the whole call, copies included, as Table 1's
 * outer times measure it).  Labels of n host-resident records (h_x: n rows of the tree's n_features floats, row
 * stride ld >= n_features floats) written to the host buffer h_out (n uint8 or int32
 * values).  Synchronous: returns when h_out is complete; the buffers are only read and
 * written during the call.  Page-locked buffers (allocated with hipHostMalloc, or
 * torch's pin_memory) are copied by DMA directly; others are staged through the
 * pipeline's pinned buffers by the host.  A pipeline serves one call at a time.
 * stats may be NULL.
 * Errors: those of dt_classify; DT_ERR_INVALID_ARG also for a null pipeline or a tree of
 * another n_features or device than the pipeline's.  On an error no copy or kernel of
 * the call is left running.
 */
dt_status dt_classify_host(const dt_tree *tree, dt_pipeline *pipeline, const float *h_x,
                           int64_t n, int64_t ld, void *h_out, dt_output out_kind,
                           dt_algo algo, dt_pipeline_stats *stats);

/* Outer-time classification (Section 4.2) of narrow records (Section 2.1's ordered
 * discrete attributes).  As dt_classify_host for records of element type x_type
 * (dt_classify_typed): h_x holds
 * elements of x_type (aligned to the element size), ld counts elements.  Narrow records
 * cross PCIe in their own width.  Errors: as dt_classify_host and dt_classify_typed. */
dt_status dt_classify_host_typed(const dt_tree *tree, dt_pipeline *pipeline, const void *h_x,
                                 dt_dtype x_type, int64_t n, int64_t ld, void *h_out,
                                 dt_output out_kind, dt_algo algo, dt_pipeline_stats *stats);

/* Outer-time classification (Section 4.2) of a forest's majority vote (Section 1): as
 * dt_classify_host for dt_forest_classify. */
dt_status dt_forest_classify_host(const dt_forest *forest, dt_pipeline *pipeline,
                                  const float *h_x, int64_t n, int64_t ld, void *h_out,
                                  dt_output out_kind, dt_algo algo, dt_pipeline_stats *stats);

/* ---- host-resident records without allocation ----------------------------------------
 *
 * For callers that cannot allocate (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): dt_classify_host for fp32 records without a pipeline.
 * The records cross to the device in chunks through a staging area that is part of the
 * library (DT_NOALLOC_SCRATCH_BYTES bytes per device, a fixed array of the library's code
 * object, held by each device the library runs on until the process ends); each chunk is
 * copied in, classified and its labels copied out, one after the other on `stream`.  The
 * call allocates no device or host memory and creates no stream or event.
 *   h_x     host records, n rows of n_features floats, row stride ld >= n_features floats
 *   h_out   host buffer of n uint8 or int32 labels (out_kind)
 *   stream  a hipStream_t of the tree's device (NULL = the null stream)
 * Synchronous: returns when h_out is complete.  Inputs of any size are processed, in chunks
 * of up to (DT_NOALLOC_SCRATCH_BYTES - 256) / (4 n_features + label bytes) records.
 * Every call on a device shares that device's staging area, which keeps the last call's
 * contents: calls that overlap on one device (from several host threads, or on several
 * streams) race and must not be made.
 * Errors: those of dt_classify_host; DT_ERR_UNSUPPORTED for a device index above 63.
 */
#define DT_NOALLOC_SCRATCH_BYTES (32 << 20)
dt_status dt_classify_host_noalloc(const dt_tree *tree, const float *h_x, int64_t n,
                                   int64_t ld, void *h_out, dt_output out_kind, dt_algo algo,
                                   void *stream);

/* Size in bytes of the per-device staging area of dt_classify_host_noalloc. */
int64_t dt_noalloc_scratch_bytes(void);

#ifdef __cplusplus
}
#endif

#endif /* DTREE_H */
