// gfx950 kernel for the literal path-reduction form of the speculative decomposition.
//
// Sections 3.3-3.4 (Procedures 4 and 5) evaluate every decision node of a record at once
// and then reduce a shared `path` array by pointer jumping: each node's entry holds the
// index of the child its predicate chose, leaf entries hold themselves (static, set once),
// and every processor repeatedly replaces its entry by the entry `hops` further along,
// until the root's entry names a leaf.  This kernel does exactly that on the same windows
// as spec_kernel (see encode.hpp): a segment of S = 2^D lanes is one record group, lane j
// is the processor of heap slot j (the processor-node map), the window's bottom positions
// S..2S-1 play the leaves (their entries point to themselves), and the reduction runs in a
// per-segment LDS array.  As in the paper's own kernel, the lanes of a wavefront execute
// in lockstep, so no workgroup barrier separates the rounds; a wavefront's LDS reads of a
// round complete before its writes.
//
// It is slower than spec_kernel, whose 64-bit predicate mask and register bit-walk need no
// path array at all; it exists to measure what that design buys over the paper's.
#include "device_common.hpp"

namespace dtree {
namespace {

using dev::Slot;

template <int RS, int D>
struct PathJump {
    static constexpr int S = 1 << D;
    int j;          // slot this lane evaluates (slot 0 is padding)
    int seg_shift;  // first lane of this lane's segment
    int *path;      // this segment's array: entries 0 .. 2S-1

    __device__ __forceinline__ PathJump(int lane, int *wave_path)
        : j(lane & (S - 1)), seg_shift(lane & ~(S - 1)),
          path(wave_path + (lane >> D) * (2 * S)) {
        // static entries: padding slot 0 and the leaves (window exits) point to themselves
        path[j + S] = j + S;
        if (j == 0) path[0] = 0;
        dev::wave_sync();
    }

    // Exit index of this lane's record for one window level.  Round g evaluates record
    // seg_shift + g in every segment; its result is kept by the lane with j == g.
    __device__ __forceinline__ int eval(const Slot *slots, bool first, const Slot &root, int w,
                                        const float *tile, int hops) const {
        int mine = 0;
        for (int g = 0; g < S; ++g) {
            const int r = seg_shift + g;
            Slot p;
            if (first) {
                p = root;
            } else {
                int wr;
                if constexpr (S == 64)
                    wr = __builtin_amdgcn_readlane(w, g);
                else
                    wr = __shfl(w, r);
                p = slots[(wr << D) + j];
            }
            const float xv = dev::feature_at<kXF32, 1>(tile + r * RS, p, dev::swz<RS>(r));
            // node evaluation: the chosen child of slot j
            if (j > 0) path[j] = 2 * j + int(!(xv < p.t));
            dev::wave_sync();
            // path reduction: entry <- entry `hops` steps further, until the root's entry
            // is a leaf; each round at least doubles the reach, so D rounds always suffice
            for (int round = 0; round < D; ++round) {
                if (__all(path[1] >= S)) break;
                int v = path[j];
                for (int h = 0; h < hops; ++h) v = path[v];
                dev::wave_sync();             // every read of this round precedes the writes
                if (j > 0) path[j] = v;
                dev::wave_sync();
            }
            const int e = path[1] - S;
            if (j == g) mine = e;
            dev::wave_sync();                 // result read before the next evaluation
        }
        return mine;
    }

    __device__ __forceinline__ int32_t run(const Slot *slots, const int32_t *exits, int levels,
                                           const Slot &root, const float *tile, int hops) const {
        int w = 0;
        int32_t code = exits[eval(slots, true, root, 0, tile, hops)];
        bool done = code < 0;
        if (!done) w = code;
        for (int level = 1; level < levels; ++level) {
            if (__all(done)) break;
            const int e = eval(slots, false, root, w, tile, hops);
            if (!done) {
                code = exits[(w << D) + e];
                done = code < 0;
                if (!done) w = code;
            }
        }
        return code;
    }
};

template <int RS, int LOAD, bool TAB_LDS, int D>
__global__ void __launch_bounds__(512) path_kernel(KArgs a) {
    extern __shared__ int4 lds[];
    const Slot *slots;
    const int32_t *exits;
    char *tiles = dev::bind_tables<TAB_LDS>(a, lds, slots, exits);
    const int lane = threadIdx.x & 63;
    float *tile;
    uint8_t *obuf;
    dev::wave_buffers<kXF32, RS>(a, tiles, tile, obuf);
    // path arrays follow the result buffers: one int per lane pair (2S per segment)
    int *wave_path = reinterpret_cast<int *>(
                         tiles + a.waves * (kTileRows * RS * 4 +
                                            out_buffer_bytes(a.out_cap, a.out_kind == 0 ? 1 : 4))) +
                     (threadIdx.x >> 6) * kPathIntsPerWave;
    const PathJump<RS, D> pj(lane, wave_path);
    const Slot root = slots[pj.j];
    dev::tile_loop<kXF32, RS, LOAD>(a, tile, obuf, lane, [&](int64_t) -> int32_t {
        return ~pj.run(slots, exits, a.levels, root, tile, a.hops);
    });
}

template <int RS, int LOAD, bool TAB_LDS>
const void *for_depth(int depth) {
    switch (depth) {
        case 1: return reinterpret_cast<const void *>(&path_kernel<RS, LOAD, TAB_LDS, 1>);
        case 2: return reinterpret_cast<const void *>(&path_kernel<RS, LOAD, TAB_LDS, 2>);
        case 3: return reinterpret_cast<const void *>(&path_kernel<RS, LOAD, TAB_LDS, 3>);
        case 4: return reinterpret_cast<const void *>(&path_kernel<RS, LOAD, TAB_LDS, 4>);
        case 5: return reinterpret_cast<const void *>(&path_kernel<RS, LOAD, TAB_LDS, 5>);
        case 6: return reinterpret_cast<const void *>(&path_kernel<RS, LOAD, TAB_LDS, 6>);
        default: return nullptr;
    }
}

template <int RS, int LOAD>
const void *for_load(bool tab_lds, int depth) {
    return tab_lds ? for_depth<RS, LOAD, true>(depth) : for_depth<RS, LOAD, false>(depth);
}

template <int RS>
const void *for_stride(int load_mode, bool tab_lds, int depth) {
    switch (load_mode) {
        case kLoadScalar: return for_load<RS, kLoadScalar>(tab_lds, depth);
        case kLoadVec: return for_load<RS, kLoadVec>(tab_lds, depth);
        case kLoadExact: return for_load<RS, kLoadExact>(tab_lds, depth);
        default: return nullptr;
    }
}

}  // namespace

const void *path_kernel_for(int row_stride, int load_mode, bool tables_in_lds, int depth) {
    switch (row_stride) {
        case 4: return for_stride<4>(load_mode, tables_in_lds, depth);
        case 8: return for_stride<8>(load_mode, tables_in_lds, depth);
        case 16: return for_stride<16>(load_mode, tables_in_lds, depth);
        case 32: return for_stride<32>(load_mode, tables_in_lds, depth);
        case 64: return for_stride<64>(load_mode, tables_in_lds, depth);
        case 128: return for_stride<128>(load_mode, tables_in_lds, depth);
        case 256: return for_stride<256>(load_mode, tables_in_lds, depth);
        default: return nullptr;
    }
}

}  // namespace dtree
