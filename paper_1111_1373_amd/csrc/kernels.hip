// gfx950 kernels for single-tree evaluation.
//
// Both kernels are persistent: each wavefront owns a private tile of 64 records in the
// LDS and walks a contiguous range of record tiles, keeping the loads of its next tile in
// flight in registers while it walks the current one, and writing its results in bursts
// from an LDS buffer.  The tree's window tables
// (see encode.hpp) are staged into the LDS once per workgroup, or, for trees whose tables
// do not fit next to the record tiles, read from global memory (L2-resident).
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

// Results of up to out_cap tiles are collected in the wavefront's LDS buffer and written in
// bursts.  Writing each tile's 64 results as soon as they are known interleaves small
// writes with the input stream, which measurably slows the stream; bursts of whole
// 16-byte vectors do not.  buf holds results of records r0 .. r0 + count - 1.
__device__ __forceinline__ void flush_results(const KArgs &a, const uint8_t *buf, int64_t r0,
                                              int64_t r_end, int lane) {
    const int esize = a.out_kind == 0 ? 1 : 4;
    const int64_t r1 = r_end < a.in.n ? r_end : a.in.n;
    const int nbytes = int(r1 - r0) * esize;
    uint8_t *dst = static_cast<uint8_t *>(a.out) + r0 * esize;
    int done = 0;
    if (a.out_vec) {   // dst is 16-byte aligned: r0 is a multiple of 64 records
        typedef int i32x4 __attribute__((ext_vector_type(4)));
        const int nvec = nbytes >> 4;
        for (int i = lane; i < nvec; i += 64)
            __builtin_nontemporal_store(reinterpret_cast<const i32x4 *>(buf)[i],
                                        reinterpret_cast<i32x4 *>(dst) + i);
        done = nvec << 4;
    }
    if (esize == 1) {
        for (int i = done + lane; i < nbytes; i += 64) dst[i] = buf[i];
    } else {
        for (int i = (done >> 2) + lane; i < (nbytes >> 2); i += 64)
            reinterpret_cast<int32_t *>(dst)[i] = reinterpret_cast<const int32_t *>(buf)[i];
    }
}

// Persistent tile loop.  Wavefront g of G takes the contiguous tile range
// [g*chunk, (g+1)*chunk), chunk = ceil(tiles / G), so its results form one contiguous run
// of the output.  `body(t)` walks staged tile t and returns each lane's result.  No
// workgroup barrier inside: the wavefronts of a workgroup process different numbers of
// tiles.
template <int RS, int LOAD, class Body>
__device__ __forceinline__ void tile_loop(const KArgs &a, float *tile, uint8_t *obuf, int lane,
                                          Body body) {
    const int64_t G = int64_t(gridDim.x) * a.waves;
    const int64_t gw = int64_t(blockIdx.x) * a.waves + (threadIdx.x >> 6);
    const int64_t chunk = (a.in.n_tiles + G - 1) / G;
    const int64_t t0 = gw * chunk < a.in.n_tiles ? gw * chunk : a.in.n_tiles;
    const int64_t t1 = t0 + chunk < a.in.n_tiles ? t0 + chunk : a.in.n_tiles;
    const int64_t n_full = a.in.n / kTileRows;     // tiles with 64 valid records
    const int esize = a.out_kind == 0 ? 1 : 4;
    int64_t fl = t0;                               // first tile whose results are buffered

    auto finish = [&](int64_t t, int32_t v) {
        const int slot = int(t - fl) * kTileRows + lane;
        if (esize == 1)
            obuf[slot] = uint8_t(v);
        else
            reinterpret_cast<int32_t *>(obuf)[slot] = v;
        if (t - fl == a.out_cap - 1 || t + 1 == t1) {
            dev::wave_sync();
            flush_results(a, obuf, fl * kTileRows, (t + 1) * kTileRows, lane);
            dev::wave_sync();
            fl = t + 1;
        }
    };

    if constexpr (LOAD != kLoadScalar && RS <= 64) {
        // Full tiles: the loads of tile t + 1 are in flight in registers while tile t is
        // walked.  The partial last tile of the input, if any, is staged on its own.
        dev::VecTile<RS, LOAD == kLoadExact> buf;
        const int64_t tf = t1 < n_full ? t1 : n_full;
        int64_t t = t0;
        if (t < tf) buf.load_full(a.in, t, lane);
        for (; t < tf; ++t) {
            dev::wave_sync();                 // previous tile fully read
            buf.store(a.in, tile, lane);
            dev::wave_sync();                 // tile visible to every lane
            if (t + 1 < tf) buf.load_full(a.in, t + 1, lane);
            finish(t, body(t));
        }
        if (t < t1) {                         // t == n_full: the partial tile
            dev::wave_sync();
            dev::stage_now<RS, LOAD>(a.in, tile, t, lane);
            dev::wave_sync();
            finish(t, body(t));
        }
    } else {
        for (int64_t t = t0; t < t1; ++t) {
            dev::wave_sync();
            dev::stage_now<RS, LOAD>(a.in, tile, t, lane);
            dev::wave_sync();
            finish(t, body(t));
        }
    }
}

// LDS layout: [tables (if staged)] [one record tile per wavefront] [one result buffer per
// wavefront].
template <int RS>
__device__ __forceinline__ void wave_buffers(const KArgs &a, char *after_tables, float *&tile,
                                             uint8_t *&obuf) {
    const int wave = threadIdx.x >> 6;
    tile = reinterpret_cast<float *>(after_tables) + wave * (kTileRows * RS);
    const int obytes = out_buffer_bytes(a.out_cap, a.out_kind == 0 ? 1 : 4);
    obuf = reinterpret_cast<uint8_t *>(after_tables) + a.waves * (kTileRows * RS * 4) + wave * obytes;
}

template <int RS, int LOAD, bool TAB_LDS>
__global__ void __launch_bounds__(512) data_kernel(KArgs a) {
    extern __shared__ int4 lds[];
    const Slot *slots;
    const int32_t *exits;
    char *tiles = bind_tables<TAB_LDS>(a, lds, slots, exits);
    const int lane = threadIdx.x & 63;
    float *tile;
    uint8_t *obuf;
    wave_buffers<RS>(a, tiles, tile, obuf);
    const float *row = tile + lane * RS;
    const int sw = dev::swz<RS>(lane);
    tile_loop<RS, LOAD>(a, tile, obuf, lane, [&](int64_t) -> int32_t {
        return ~dev::walk_data(slots, exits, a.depth, a.levels, row, sw);
    });
}

template <int RS, int LOAD, bool TAB_LDS, int D>
__global__ void __launch_bounds__(512) spec_kernel(KArgs a) {
    extern __shared__ int4 lds[];
    const Slot *slots;
    const int32_t *exits;
    char *tiles = bind_tables<TAB_LDS>(a, lds, slots, exits);
    const int lane = threadIdx.x & 63;
    float *tile;
    uint8_t *obuf;
    wave_buffers<RS>(a, tiles, tile, obuf);
    const dev::Spec<RS, D> spec(lane);
    const Slot root = slots[spec.j];   // window 0 is shared by every record
    tile_loop<RS, LOAD>(a, tile, obuf, lane, [&](int64_t) -> int32_t {
        return ~spec.run(slots, exits, a.levels, root, tile);
    });
}

// ---- instance tables ------------------------------------------------------------------
template <int RS, int LOAD, bool TAB_LDS>
const void *spec_for(int depth) {
    switch (depth) {
        case 1: return reinterpret_cast<const void *>(&spec_kernel<RS, LOAD, TAB_LDS, 1>);
        case 2: return reinterpret_cast<const void *>(&spec_kernel<RS, LOAD, TAB_LDS, 2>);
        case 3: return reinterpret_cast<const void *>(&spec_kernel<RS, LOAD, TAB_LDS, 3>);
        case 4: return reinterpret_cast<const void *>(&spec_kernel<RS, LOAD, TAB_LDS, 4>);
        case 5: return reinterpret_cast<const void *>(&spec_kernel<RS, LOAD, TAB_LDS, 5>);
        case 6: return reinterpret_cast<const void *>(&spec_kernel<RS, LOAD, TAB_LDS, 6>);
        default: return nullptr;
    }
}

template <int RS, int LOAD, bool TAB_LDS>
const void *for_variant(int algo, int depth) {
    if (algo == kAlgoData) return reinterpret_cast<const void *>(&data_kernel<RS, LOAD, TAB_LDS>);
    return spec_for<RS, LOAD, TAB_LDS>(depth);
}

template <int RS, int LOAD>
const void *for_load(int algo, bool tab_lds, int depth) {
    return tab_lds ? for_variant<RS, LOAD, true>(algo, depth)
                   : for_variant<RS, LOAD, false>(algo, depth);
}

template <int RS>
const void *for_stride(int algo, int load_mode, bool tab_lds, int depth) {
    switch (load_mode) {
        case kLoadScalar: return for_load<RS, kLoadScalar>(algo, tab_lds, depth);
        case kLoadVec: return for_load<RS, kLoadVec>(algo, tab_lds, depth);
        case kLoadExact: return for_load<RS, kLoadExact>(algo, tab_lds, depth);
        default: return nullptr;
    }
}

}  // namespace

const void *kernel_for(int algo, int row_stride, int load_mode, bool tables_in_lds, int depth) {
    switch (row_stride) {
        case 4: return for_stride<4>(algo, load_mode, tables_in_lds, depth);
        case 8: return for_stride<8>(algo, load_mode, tables_in_lds, depth);
        case 16: return for_stride<16>(algo, load_mode, tables_in_lds, depth);
        case 32: return for_stride<32>(algo, load_mode, tables_in_lds, depth);
        case 64: return for_stride<64>(algo, load_mode, tables_in_lds, depth);
        case 128: return for_stride<128>(algo, load_mode, tables_in_lds, depth);
        case 256: return for_stride<256>(algo, load_mode, tables_in_lds, depth);
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
