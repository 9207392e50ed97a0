// gfx950 kernels for single-tree evaluation, templated on the record element type.  Each
// element type is instantiated in a translation unit of its own (kernels.hip: fp32,
// kernels_f16.hip, kernels_bf16.hip, kernels_u8.hip).
//
// Both kernels are persistent: each wavefront owns a private tile of 64 records in the
// LDS and walks a contiguous range of record tiles, keeping the loads of its next tile in
// flight in registers while it walks the current one, and writing its results in bursts
// from an LDS buffer.  The tree's window tables (see encode.hpp) are staged into the LDS
// once per workgroup, or, for trees whose tables do not fit next to the record tiles, read
// from global memory (L2-resident).  Records stay in their own element type in the LDS;
// every tree step widens the element it reads to fp32 and compares it with the fp32
// threshold, which is the decision on the stored value.
//
//   data_kernel  (Section 3.2, Procedure 3): lane r evaluates record r of its tile.
//   spec_kernel  (Sections 3.3-3.4, Procedures 4-5): 2^D lanes evaluate all slots of a
//                record's current window at once; a wavefront ballot gathers the outcomes
//                and the exit is found by walking the bits.  The mask replaces the paper's
//                shared `path` array and its barrier-separated pointer jumping.
#pragma once

#include "device_common.hpp"

namespace dtree {
namespace {

using dev::Slot;

template <int XT, int RS, int LOAD, bool TAB_LDS>
__global__ void __launch_bounds__(512) data_kernel(KArgs a) {
    using T = typename dev::Elem<XT>::T;
    extern __shared__ int4 lds[];
    const typename dev::Node<XT>::S *slots;
    const int32_t *exits;
    char *tiles = dev::bind_tables<TAB_LDS>(a, lds, slots, exits);
    const int lane = threadIdx.x & 63;
    float *tile;
    uint8_t *obuf;
    dev::wave_buffers<XT, RS>(a, tiles, tile, obuf);
    const T *row = reinterpret_cast<const T *>(tile) + lane * RS;
    const int sw = dev::swz_el<XT, RS>(lane);
    const typename dev::Node<XT>::S root0 = slots[1];   // window 0's root, for every record
    dev::tile_loop<XT, RS, LOAD>(a, tile, obuf, lane, [&](int64_t) -> int32_t {
        return ~dev::walk_data<XT>(slots, exits, a.depth, a.levels, row, sw, root0);
    });
}

template <int XT, int RS, int LOAD, bool TAB_LDS, int D>
__global__ void __launch_bounds__(64 * tree_max_waves(kAlgoSpec, D, RS * int(sizeof(typename dev::Elem<XT>::T))))
spec_kernel(KArgs a) {
    using T = typename dev::Elem<XT>::T;
    using NS = typename dev::Node<XT>::S;
    extern __shared__ int4 lds[];
    const NS *slots;
    const int32_t *exits;
    char *tiles = dev::bind_tables<TAB_LDS>(a, lds, slots, exits);
    const int lane = threadIdx.x & 63;
    constexpr int TR = tile_rows_for(kAlgoSpec, D, RS * int(sizeof(T)));
    float *tile;
    uint8_t *obuf;
    dev::wave_buffers<XT, RS, TR>(a, tiles, tile, obuf);
    using Spec = dev::Spec<XT, RS, D, TR>;
    const Spec spec(lane);
    const NS root = slots[spec.j];   // window 0 is shared by every record
    const T *el = reinterpret_cast<const T *>(tile);
    dev::tile_loop<XT, RS, LOAD, Spec::kLayout, TR>(a, tile, obuf, lane, [&](int64_t) -> int32_t {
        return ~spec.in_record_order(spec.run(slots, exits, a.levels, root, el));
    });
}

// ---- instance tables ------------------------------------------------------------------
template <int XT, int RS, int LOAD, bool TAB_LDS>
const void *spec_for(int depth) {
    switch (depth) {
        case 1: return reinterpret_cast<const void *>(&spec_kernel<XT, RS, LOAD, TAB_LDS, 1>);
        case 2: return reinterpret_cast<const void *>(&spec_kernel<XT, RS, LOAD, TAB_LDS, 2>);
        case 3: return reinterpret_cast<const void *>(&spec_kernel<XT, RS, LOAD, TAB_LDS, 3>);
        case 4: return reinterpret_cast<const void *>(&spec_kernel<XT, RS, LOAD, TAB_LDS, 4>);
        case 5: return reinterpret_cast<const void *>(&spec_kernel<XT, RS, LOAD, TAB_LDS, 5>);
        case 6: return reinterpret_cast<const void *>(&spec_kernel<XT, RS, LOAD, TAB_LDS, 6>);
        default: return nullptr;
    }
}

template <int XT, int RS, int LOAD, bool TAB_LDS>
const void *for_variant(int algo, int depth) {
    if (algo == kAlgoData)
        return reinterpret_cast<const void *>(&data_kernel<XT, RS, LOAD, TAB_LDS>);
    if (algo == kAlgoSpec) return spec_for<XT, RS, LOAD, TAB_LDS>(depth);
    return nullptr;
}

template <int XT, int RS, int LOAD>
const void *for_load(int algo, bool tab_lds, int depth) {
    if constexpr (LOAD != kLoadScalar && !dev::has_vec_staging<XT, RS>()) {
        return nullptr;   // rows narrower than one 16-byte vector: scalar loads only
    } else {
        return tab_lds ? for_variant<XT, RS, LOAD, true>(algo, depth)
                       : for_variant<XT, RS, LOAD, false>(algo, depth);
    }
}

template <int XT, int RS>
const void *for_stride(int algo, int load_mode, bool tab_lds, int depth) {
    switch (load_mode) {
        case kLoadScalar: return for_load<XT, RS, kLoadScalar>(algo, tab_lds, depth);
        case kLoadVec: return for_load<XT, RS, kLoadVec>(algo, tab_lds, depth);
        case kLoadExact: return for_load<XT, RS, kLoadExact>(algo, tab_lds, depth);
        default: return nullptr;
    }
}

template <int XT>
const void *single_tree_kernel(int algo, int row_stride, int load_mode, bool tab_lds, int depth) {
    switch (row_stride) {
        case 4: return for_stride<XT, 4>(algo, load_mode, tab_lds, depth);
        case 8: return for_stride<XT, 8>(algo, load_mode, tab_lds, depth);
        case 16: return for_stride<XT, 16>(algo, load_mode, tab_lds, depth);
        case 32: return for_stride<XT, 32>(algo, load_mode, tab_lds, depth);
        case 64: return for_stride<XT, 64>(algo, load_mode, tab_lds, depth);
        case 128: return for_stride<XT, 128>(algo, load_mode, tab_lds, depth);
        case 256: return for_stride<XT, 256>(algo, load_mode, tab_lds, depth);
        default: return nullptr;
    }
}

}  // namespace
}  // namespace dtree
