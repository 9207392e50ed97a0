// Interface between the host library (dtree.hip) and the gfx950 kernels (kernels.hip).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace dtree {

constexpr int kTileRows = 64;          // records per wavefront tile (one per lane)
constexpr int kMaxRowStride = 256;     // LDS row stride limit in floats (n_features <= 256)
constexpr int kMaxWavesPerBlock = 8;   // kernels are built for <= 512 threads
constexpr int kMaxForestTrees = 255;   // 8-bit vote counters
constexpr int kMaxForestClasses = 64;  // 16 VGPRs of packed counters

// The record matrix a kernel reads.
struct Rows {
    const float *x;          // device features, row-major
    int64_t n;               // records
    int64_t ld;              // row stride in floats
    int64_t n_tiles;         // ceil(n / 64)
    int32_t n_features;      // F
    uint32_t magic_f;        // ceil(2^32 / F) for F >= 2 (row = idx / F via mulhi)
};

// Single-tree kernel arguments (passed by value).
struct KArgs {
    Rows in;
    const int4 *slots;       // n_slots (threshold, feature) pairs, 8 bytes each
    const int4 *exits;       // n_slots int32 exit codes
    int32_t slot_bytes;      // bytes of the slot region (multiple of 16)
    int32_t exit_bytes;      // bytes of the exit region (multiple of 16)
    int32_t depth;           // window depth D
    int32_t levels;          // windows on the longest path
    int32_t waves;           // wavefronts per workgroup
    int32_t out_kind;        // 0: uint8 output, 1: int32 output
    int32_t out_cap;         // tiles of results each wavefront buffers in the LDS (>= 1)
    int32_t out_vec;         // 1: `out` is 16-byte aligned (flushes use 16-byte stores)
    int32_t hops;            // path-reduction kernel: further entries read per round
    void *out;
};

// Path-reduction kernel: per wavefront, 64/S segments of 2S path entries (S lanes each).
constexpr int kPathIntsPerWave = 128;

// LDS bytes of one wavefront's result buffer: cap tiles of 64 results of out_bytes each.
__host__ __device__ inline int out_buffer_bytes(int cap, int out_bytes) { return cap * kTileRows * out_bytes; }

// Forest kernel arguments.  Tree k's tables are the bytes [off_k, off_k + slot_bytes_k)
// (slots) followed by its exit codes, inside `tables`; trees[k] = {off_k, slot_bytes_k,
// levels_k, 0}.  Chunks are runs of consecutive trees staged into the LDS together:
// chunks[c] = {first_tree, end_tree, byte_off, bytes}.
struct FArgs {
    Rows in;
    const int4 *tables;
    const int4 *trees;
    const int4 *chunks;
    int32_t n_trees;
    int32_t n_chunks;
    int32_t table_lds_bytes; // LDS bytes reserved for one chunk (0: tables read in place)
    int32_t depth;           // window depth D (every tree)
    int32_t n_classes;
    int32_t waves;
    int32_t out_kind;        // 0: uint8 output, 1: int32 output
    void *out;
};

enum KernelAlgo { kAlgoData = 0, kAlgoSpec = 1, kAlgoPath = 2 };

// How record tiles are read from HBM.
enum LoadMode {
    kLoadScalar = 0,   // any ld >= F, 4-byte aligned: one float per load
    kLoadVec = 1,      // ld == F, F % 4 == 0, 16-byte aligned base: 16-byte loads
    kLoadExact = 2,    // as kLoadVec and F == the LDS row stride: every lane loads RS/4
                       // vectors per tile with no bounds test
    kLoadModes = 3
};

// Kernel instance for (algorithm, LDS row stride, load mode, tables staged in the LDS or
// read from global memory, window depth), or nullptr if no such instance exists.
// `depth` is ignored by the data kernel.
const void *kernel_for(int algo, int row_stride, int load_mode, bool tables_in_lds, int depth);

// Path-reduction kernel instance (speculative windows of depth 1..6).
const void *path_kernel_for(int row_stride, int load_mode, bool tables_in_lds, int depth);

// Forest kernel instance; `vote_words` = 32-bit words of packed 8-bit counters
// (2, 4 or 16 for up to 8, 16 or 64 classes).
const void *forest_kernel_for(int algo, int row_stride, int load_mode, bool tables_in_lds,
                              int vote_words, int depth);

// One-time per-instance setup (raise the dynamic LDS limit to the device maximum).
hipError_t prepare_kernel(const void *fn, int max_lds_bytes);

// Launches: grid of `blocks` workgroups of args.waves wavefronts.
hipError_t launch_kernel(const void *fn, const KArgs &args, int blocks, int lds_bytes,
                         hipStream_t stream);
hipError_t launch_forest(const void *fn, const FArgs &args, int blocks, int lds_bytes,
                         hipStream_t stream);

// Dynamic LDS of a workgroup of `waves` wavefronts: tables, one record tile per wavefront,
// then (single-tree kernels) one result buffer of `out_bytes_per_wave` per wavefront.
inline int lds_bytes_for(int table_bytes, int row_stride, int waves, int out_bytes_per_wave = 0) {
    return table_bytes + waves * (kTileRows * row_stride * 4 + out_bytes_per_wave);
}

}  // namespace dtree
