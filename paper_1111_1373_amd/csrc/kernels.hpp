// Interface between the host library (dtree.hip) and the gfx950 kernels (kernels.hip).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace dtree {

enum KernelAlgo { kAlgoData = 0, kAlgoSpec = 1, kAlgoPath = 2 };

constexpr int kTileRows = 64;          // records per wavefront tile (one per lane)
constexpr int kMaxRowStride = 256;     // LDS row stride limit in floats (n_features <= 256)
constexpr int kMaxWavesPerBlock = 8;   // kernels are built for <= 512 threads, except:
// forest instances whose registers fit 16 wavefronts per CU without spilling (data walk
// on rows of up to 128 features, speculative walk with depth-2 windows on rows of up to
// 32), built for <= 1024.  `depth` is the speculative window depth (unused for data).
constexpr int kMaxForestWavesPerBlock = 16;
__host__ __device__ constexpr int forest_max_waves(int algo, int depth, int row_stride) {
    return (algo == 0 ? row_stride <= 128 : depth == 2 && row_stride <= 32)
               ? kMaxForestWavesPerBlock
               : kMaxWavesPerBlock;
}
constexpr int kMaxForestTrees = 255;   // 8-bit vote counters
constexpr int kMaxForestClasses = 64;  // 16 VGPRs of packed counters

// Record element types (values of dt_dtype).  Each widens exactly to fp32.
enum ElemType { kXF32 = 0, kXF16 = 1, kXBF16 = 2, kXU8 = 3, kElemTypes = 4 };

__host__ __device__ inline int elem_bytes(int xt) { return xt == kXF32 ? 4 : xt == kXU8 ? 1 : 2; }

// The record matrix a kernel reads.
struct Rows {
    const void *x;           // device records, row-major, elements of the kernel's type
    int64_t n;               // records
    int64_t ld;              // row stride in elements
    int64_t n_tiles;         // ceil(n / 64)
    int32_t n_features;      // F
    uint32_t magic_f;        // ceil(2^32 / F) for F >= 2 (row = idx / F via mulhi)
    int32_t n_words;         // 4-byte words per dense row, F * elem_bytes / 4 (vector loads)
    uint32_t magic_w;        // ceil(2^32 / n_words) for n_words >= 2
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

// Records per wavefront tile of a kernel: 64 (one per lane), except for the speculative
// kernel with 32- and 64-slot windows (depths 5 and 6) on rows of at least 32 bytes in the
// LDS.  That kernel reads one or two record rows per round, so a tile of 32 records serves
// it as well while taking half the LDS, and twice as many wavefronts then fit next to its
// window tables.  (Rows under 32 bytes keep 64 records: 16-byte staging needs one vector
// per lane.)
__host__ __device__ constexpr int tile_rows_for(int algo, int depth, int row_bytes) {
    return algo == kAlgoSpec && depth >= 5 && row_bytes >= 32 ? 32 : kTileRows;
}

// Largest workgroup of a single-tree kernel instance, in wavefronts: 8, or 16 for the
// speculative walk on 32-record tiles, whose registers (at most 128 per lane) fit 16
// wavefronts per CU and whose small tiles leave the LDS room for them.
__host__ __device__ constexpr int tree_max_waves(int algo, int depth, int row_bytes) {
    return tile_rows_for(algo, depth, row_bytes) < kTileRows ? 16 : kMaxWavesPerBlock;
}

// LDS bytes of one wavefront's result buffer: cap tiles of `tile_rows` results of
// out_bytes each.
__host__ __device__ inline int out_buffer_bytes(int cap, int out_bytes, int tile_rows = kTileRows) {
    return cap * tile_rows * out_bytes;
}

// Forest kernel arguments.  Tree k's tables are the bytes [off_k, off_k + slot_bytes_k)
// (slots) followed by its exit codes (int16 when every code of the forest fits, else
// int32), inside `tables`; trees[k] = {off_k, slot_bytes_k, levels_k, 0}.  Chunks are runs of consecutive trees staged into the LDS together:
// chunks[c] = {first_tree, end_tree, byte_off, bytes}.
struct FArgs {
    Rows in;
    const int4 *tables;
    const int4 *trees;
    const int2 *roots;       // per tree: the root slot {threshold bits, feature byte offset}
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

// How record tiles are read from HBM.
enum LoadMode {
    kLoadScalar = 0,   // any ld >= F, element-aligned: one element per load
    kLoadVec = 1,      // ld == F, F * elem_bytes % 16 == 0, 16-byte aligned base: 16-byte loads
    kLoadExact = 2,    // as kLoadVec and F == the LDS row stride: every lane loads the same
                       // number of vectors per tile with no bounds test
    kLoadModes = 3
};

// Kernel instance for (algorithm, record element type, LDS row stride in elements, load
// mode, tables staged in the LDS or read from global memory, window depth), or nullptr if
// no such instance exists.  `depth` is ignored by the data kernel.
const void *kernel_for(int algo, int elem_type, int row_stride, int load_mode, bool tables_in_lds,
                       int depth);

// Per element type (one translation unit each): data and speculative kernel instances.
const void *kernel_for_f32(int algo, int row_stride, int load_mode, bool tables_in_lds, int depth);
const void *kernel_for_f16(int algo, int row_stride, int load_mode, bool tables_in_lds, int depth);
const void *kernel_for_bf16(int algo, int row_stride, int load_mode, bool tables_in_lds, int depth);
const void *kernel_for_u8(int algo, int row_stride, int load_mode, bool tables_in_lds, int depth);

// Path-reduction kernel instance (fp32 records, speculative windows of depth 1..6).
const void *path_kernel_for(int row_stride, int load_mode, bool tables_in_lds, int depth);

// Forest kernel instance; `vote_words` = 32-bit words of packed 8-bit counters
// (2, 4 or 16 for up to 8, 16 or 64 classes); `exit_mode`: exit codes stored as int32 (0)
// or int16 (1) tables, or packed into the windows' bottom slots (2, data walk only).
const void *forest_kernel_for(int algo, int row_stride, int load_mode, bool tables_in_lds,
                              int vote_words, int depth, int exit_mode);
// The int16 and the packed instances (translation units of their own).
const void *forest_kernel_for_ex16(int algo, int row_stride, int load_mode, bool tables_in_lds,
                                   int vote_words, int depth);
const void *forest_kernel_for_packed(int algo, int row_stride, int load_mode,
                                     bool tables_in_lds, int vote_words, int depth);

// One-time per-instance setup (raise the dynamic LDS limit to the device maximum).
hipError_t prepare_kernel(const void *fn, int max_lds_bytes);

// Launches: grid of `blocks` workgroups of args.waves wavefronts.
hipError_t launch_kernel(const void *fn, const KArgs &args, int blocks, int lds_bytes,
                         hipStream_t stream);
hipError_t launch_forest(const void *fn, const FArgs &args, int blocks, int lds_bytes,
                         hipStream_t stream);

// LDS bytes of one record tile: tile_rows rows of `row_stride` elements of `elem_type`.
inline int tile_bytes_for(int row_stride, int elem_type, int tile_rows = kTileRows) {
    return tile_rows * row_stride * elem_bytes(elem_type);
}

// Dynamic LDS of a workgroup of `waves` wavefronts: tables, one record tile per wavefront,
// then (single-tree kernels) one result buffer of `out_bytes_per_wave` per wavefront.
inline int lds_bytes_for(int table_bytes, int tile_bytes, int waves, int out_bytes_per_wave = 0) {
    return table_bytes + waves * (tile_bytes + out_bytes_per_wave);
}

}  // namespace dtree
