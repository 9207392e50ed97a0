// gfx950 kernels for single-tree evaluation.
//
// Both kernels are persistent: each wavefront owns a private tile of 64 records in the
// LDS and strides over the record tiles of the whole input, prefetching the next tile into
// registers while it walks the current one.  The tree's window tables (see encode.hpp)
// are staged into the LDS once per workgroup, or, for trees whose tables do not fit next
// to the record tiles, read from global memory (L2-resident).
//
//   data_kernel  (Section 3.2, Procedure 3): lane r evaluates record r of its tile.
//   spec_kernel  (Sections 3.3-3.4, Procedures 4-5): 2^D lanes evaluate all slots of a
//                record's current window at once; a wavefront ballot gathers the outcomes
//                and the exit is found by walking the bits.  The mask replaces the paper's
//                shared `path` array and its barrier-separated pointer jumping.
#include "device_common.hpp"

namespace dtree {
namespace {

using dev::Slot;

// Window tables: staged into the LDS once per workgroup (TAB_LDS), or read in place from
// global memory.  Returns the first LDS byte after the tables (where record tiles start).
template <bool TAB_LDS>
__device__ __forceinline__ char *bind_tables(const KArgs &a, int4 *lds, const Slot *&slots,
                                             const int32_t *&exits) {
    if constexpr (TAB_LDS) {
        const int ns = a.slot_bytes >> 4;
        const int ne = a.exit_bytes >> 4;
        for (int i = threadIdx.x; i < ns; i += blockDim.x) lds[i] = a.slots[i];
        for (int i = threadIdx.x; i < ne; i += blockDim.x) lds[ns + i] = a.exits[i];
        __syncthreads();
        slots = reinterpret_cast<const Slot *>(lds);
        exits = reinterpret_cast<const int32_t *>(reinterpret_cast<const char *>(lds) + a.slot_bytes);
        return reinterpret_cast<char *>(lds) + a.slot_bytes + a.exit_bytes;
    } else {
        slots = reinterpret_cast<const Slot *>(a.slots);
        exits = reinterpret_cast<const int32_t *>(a.exits);
        return reinterpret_cast<char *>(lds);
    }
}

// Persistent tile loop; `body(t)` evaluates staged tile t.  No workgroup barrier inside:
// the wavefronts of a workgroup process different numbers of tiles.
template <int RS, bool VEC, class Body>
__device__ __forceinline__ void tile_loop(const KArgs &a, float *tile, int lane, Body body) {
    const int64_t stride = int64_t(gridDim.x) * a.waves;
    int64_t t = int64_t(blockIdx.x) * a.waves + (threadIdx.x >> 6);
    if constexpr (VEC && RS <= 64) {
        dev::VecTile<RS> buf;
        if (t < a.in.n_tiles) buf.load(a.in, t, lane);
        for (; t < a.in.n_tiles; t += stride) {
            dev::wave_sync();                 // previous tile fully read
            buf.store(a.in, tile, lane);
            dev::wave_sync();                 // tile visible to every lane
            if (t + stride < a.in.n_tiles) buf.load(a.in, t + stride, lane);   // prefetch
            body(t);
        }
    } else {
        for (; t < a.in.n_tiles; t += stride) {
            dev::wave_sync();
            dev::stage_now<RS, VEC>(a.in, tile, t, lane);
            dev::wave_sync();
            body(t);
        }
    }
}

template <int RS, bool VEC, bool TAB_LDS>
__global__ void __launch_bounds__(512) data_kernel(KArgs a) {
    extern __shared__ int4 lds[];
    const Slot *slots;
    const int32_t *exits;
    char *tiles = bind_tables<TAB_LDS>(a, lds, slots, exits);
    const int lane = threadIdx.x & 63;
    float *tile = reinterpret_cast<float *>(tiles) + (threadIdx.x >> 6) * (kTileRows * RS);
    const float *row = tile + lane * RS;
    const int sw = dev::swz<RS>(lane);
    tile_loop<RS, VEC>(a, tile, lane, [&](int64_t t) {
        const int32_t code = dev::walk_data(slots, exits, a.depth, a.levels, row, sw);
        dev::store_value(a.out, a.out_kind, a.in.n, t * kTileRows + lane, ~code);
    });
}

template <int RS, bool VEC, bool TAB_LDS, int D>
__global__ void __launch_bounds__(512) spec_kernel(KArgs a) {
    extern __shared__ int4 lds[];
    const Slot *slots;
    const int32_t *exits;
    char *tiles = bind_tables<TAB_LDS>(a, lds, slots, exits);
    const int lane = threadIdx.x & 63;
    float *tile = reinterpret_cast<float *>(tiles) + (threadIdx.x >> 6) * (kTileRows * RS);
    const dev::Spec<RS, D> spec(lane);
    const Slot root = slots[spec.j];   // window 0 is shared by every record
    tile_loop<RS, VEC>(a, tile, lane, [&](int64_t t) {
        const int32_t code = spec.run(slots, exits, a.levels, root, tile);
        dev::store_value(a.out, a.out_kind, a.in.n, t * kTileRows + lane, ~code);
    });
}

// ---- instance tables ------------------------------------------------------------------
template <int RS, bool VEC, bool TAB_LDS>
const void *spec_for(int depth) {
    switch (depth) {
        case 1: return reinterpret_cast<const void *>(&spec_kernel<RS, VEC, TAB_LDS, 1>);
        case 2: return reinterpret_cast<const void *>(&spec_kernel<RS, VEC, TAB_LDS, 2>);
        case 3: return reinterpret_cast<const void *>(&spec_kernel<RS, VEC, TAB_LDS, 3>);
        case 4: return reinterpret_cast<const void *>(&spec_kernel<RS, VEC, TAB_LDS, 4>);
        case 5: return reinterpret_cast<const void *>(&spec_kernel<RS, VEC, TAB_LDS, 5>);
        case 6: return reinterpret_cast<const void *>(&spec_kernel<RS, VEC, TAB_LDS, 6>);
        default: return nullptr;
    }
}

template <int RS, bool VEC, bool TAB_LDS>
const void *for_variant(int algo, int depth) {
    if (algo == kAlgoData) return reinterpret_cast<const void *>(&data_kernel<RS, VEC, TAB_LDS>);
    return spec_for<RS, VEC, TAB_LDS>(depth);
}

template <int RS>
const void *for_stride(int algo, bool vec, bool tab_lds, int depth) {
    if (vec)
        return tab_lds ? for_variant<RS, true, true>(algo, depth)
                       : for_variant<RS, true, false>(algo, depth);
    return tab_lds ? for_variant<RS, false, true>(algo, depth)
                   : for_variant<RS, false, false>(algo, depth);
}

}  // namespace

const void *kernel_for(int algo, int row_stride, bool vec, bool tables_in_lds, int depth) {
    switch (row_stride) {
        case 4: return for_stride<4>(algo, vec, tables_in_lds, depth);
        case 8: return for_stride<8>(algo, vec, tables_in_lds, depth);
        case 16: return for_stride<16>(algo, vec, tables_in_lds, depth);
        case 32: return for_stride<32>(algo, vec, tables_in_lds, depth);
        case 64: return for_stride<64>(algo, vec, tables_in_lds, depth);
        case 128: return for_stride<128>(algo, vec, tables_in_lds, depth);
        case 256: return for_stride<256>(algo, vec, tables_in_lds, depth);
        default: return nullptr;
    }
}

hipError_t prepare_kernel(const void *fn, int max_lds_bytes) {
    return hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, max_lds_bytes);
}

hipError_t launch_kernel(const void *fn, const KArgs &args, int blocks, int lds_bytes,
                         hipStream_t stream) {
    KArgs a = args;
    void *params[] = {&a};
    return hipLaunchKernel(fn, dim3(unsigned(blocks)), dim3(unsigned(args.waves * 64)), params,
                           size_t(lds_bytes), stream);
}

}  // namespace dtree
