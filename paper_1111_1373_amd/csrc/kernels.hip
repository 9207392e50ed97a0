// gfx950 kernels for classification-tree evaluation.
//
// Both kernels are persistent: each wavefront owns a private tile of 64 records in the
// LDS and strides over the record tiles of the whole input.  The tree's window tables
// (see encode.hpp) are staged into the LDS once per workgroup, or, for trees whose tables
// do not fit next to the record tiles, read from global memory (L2-resident).
//
//   data_kernel  (Section 3.2, Procedure 3): lane r of a wavefront evaluates record r of
//                the tile.  Within a window the walk is branch-free heap arithmetic,
//                h <- 2h + 1 + !(x[f_h] < t_h), for exactly D steps; the exit slot then
//                names the next window or the record's class.
//   spec_kernel  (Sections 3.3-3.4, Procedures 4-5): a segment of S = 2^D lanes is the
//                record group of one record; lane j evaluates heap slot j of the
//                record's current window (the processor-node map), so one wavefront
//                instruction evaluates 64/S records' windows at once.  The 64 outcomes
//                form a wavefront mask (one v_cmp writes it), the segment belonging to
//                record r is handed to lane r, and lane r finds the exit by walking its
//                own bits from the window root.  This replaces the paper's shared
//                `path` array and its barrier-separated pointer jumping, which the
//                mask makes unnecessary.
//
// Tile layout in the LDS: row r (record) at r*RS floats, column c stored at position
// c ^ swz(r).  The XOR spreads the 64 rows over all 64 banks for a fixed column, so the
// top levels of the tree (where every lane reads the same feature) are conflict-free,
// and the 16-byte staging stores land on distinct banks.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>

#include "kernels.hpp"

namespace dtree {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

struct alignas(8) Slot {
    float t;
    int32_t f;
};

template <int RS>
__device__ __forceinline__ int swz(int r) {
    if constexpr (RS >= 64) {
        return r;                                  // r < 64 <= RS
    } else {
        constexpr int sh = __builtin_ctz(64 / RS);
        return (r >> sh) & (RS - 1);
    }
}

// Ordering of LDS accesses among the lanes of one wavefront.  A wavefront's LDS
// instructions execute in order; the fences keep the compiler from moving accesses
// across this point.  No workgroup barrier is used inside the persistent loop because
// wavefronts of a workgroup process different numbers of tiles.
__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ uint32_t div_f(uint32_t e, const KArgs &a) {
    return a.n_features == 1 ? e : __umulhi(e, a.magic_f);
}

// Window tables: staged into the LDS once per workgroup (TAB_LDS), or read in place from
// global memory through the vector caches when they are too large for the LDS.
// Returns the first LDS byte after the tables (where the record tiles start).
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

// ---- staging, vectorised path: ld == F, F % 4 == 0, 16-byte aligned rows -------------
template <int RS>
struct VecTile {
    static constexpr int kVec = RS / 4;   // 16-byte vectors per lane for a full tile of F == RS
    f32x4 v[kVec];

    __device__ __forceinline__ void load(const KArgs &a, int64_t tile, int lane) {
        const int64_t row0 = tile * kTileRows;
        const int64_t rows_left = a.n - row0;
        const int valid = rows_left < kTileRows ? int(rows_left) : kTileRows;
        const int nvec = (valid * a.n_features) >> 2;
        const f32x4 *src = reinterpret_cast<const f32x4 *>(a.x + row0 * a.n_features);
#pragma unroll
        for (int k = 0; k < kVec; ++k) {
            const int q = k * 64 + lane;
            v[k] = q < nvec ? __builtin_nontemporal_load(src + q) : f32x4{0.f, 0.f, 0.f, 0.f};
        }
    }

    __device__ __forceinline__ void store(const KArgs &a, float *tile, int lane) const {
        const int full = kTileRows * a.n_features / 4;
#pragma unroll
        for (int k = 0; k < kVec; ++k) {
            const int q = k * 64 + lane;
            if (q < full) {
                const uint32_t e = uint32_t(q) * 4u;
                const int r = int(div_f(e, a));
                const int c = int(e) - r * a.n_features;
                float *row = tile + r * RS;
                const int s = swz<RS>(r);
                row[(c + 0) ^ s] = v[k].x;
                row[(c + 1) ^ s] = v[k].y;
                row[(c + 2) ^ s] = v[k].z;
                row[(c + 3) ^ s] = v[k].w;
            }
        }
    }
};

// ---- staging, general path: any ld >= F, any alignment --------------------------------
template <int RS>
__device__ __forceinline__ void stage_scalar(const KArgs &a, float *tile, int64_t tile_idx,
                                             int lane) {
    const int64_t row0 = tile_idx * kTileRows;
    const int64_t rows_left = a.n - row0;
    const int valid = rows_left < kTileRows ? int(rows_left) : kTileRows;
    for (int k = 0; k < a.n_features; ++k) {
        const uint32_t idx = uint32_t(k * 64 + lane);
        const int r = int(div_f(idx, a));
        const int c = int(idx) - r * a.n_features;
        float v = 0.f;
        if (r < valid) v = a.x[(row0 + r) * a.ld + c];
        tile[r * RS + (c ^ swz<RS>(r))] = v;
    }
}

__device__ __forceinline__ void store_out(const KArgs &a, int64_t row, int32_t code) {
    if (row < a.n) {
        const int32_t v = ~code;   // code = -(value + 1)
        if (a.out_kind == 0)
            static_cast<uint8_t *>(a.out)[row] = uint8_t(v);
        else
            static_cast<int32_t *>(a.out)[row] = v;
    }
}

// Persistent tile loop shared by both kernels; `Body(tile, lane, tile_idx)` evaluates
// one staged tile.
template <int RS, bool VEC, class Body>
__device__ __forceinline__ void tile_loop(const KArgs &a, float *tile, int lane, Body body) {
    const int64_t stride = int64_t(gridDim.x) * a.waves;
    int64_t t = int64_t(blockIdx.x) * a.waves + (threadIdx.x >> 6);
    if constexpr (VEC && RS <= 64) {
        VecTile<RS> buf;
        if (t < a.n_tiles) buf.load(a, t, lane);
        for (; t < a.n_tiles; t += stride) {
            wave_sync();                 // previous tile fully read
            buf.store(a, tile, lane);
            wave_sync();                 // tile visible to every lane
            if (t + stride < a.n_tiles) buf.load(a, t + stride, lane);   // prefetch
            body(t);
        }
    } else if constexpr (VEC) {
        for (; t < a.n_tiles; t += stride) {
            wave_sync();
            // wide rows: stage in register chunks of 16 float4 per lane, no prefetch
            const int64_t row0 = t * kTileRows;
            const int64_t rows_left = a.n - row0;
            const int valid = rows_left < kTileRows ? int(rows_left) : kTileRows;
            const int nvec = (valid * a.n_features) >> 2;
            const int full = kTileRows * a.n_features / 4;
            const f32x4 *src = reinterpret_cast<const f32x4 *>(a.x + row0 * a.n_features);
#pragma unroll 1
            for (int k0 = 0; k0 < RS / 4; k0 += 16) {
                f32x4 v[16];
#pragma unroll
                for (int k = 0; k < 16; ++k) {
                    const int q = (k0 + k) * 64 + lane;
                    v[k] = q < nvec ? __builtin_nontemporal_load(src + q) : f32x4{0.f, 0.f, 0.f, 0.f};
                }
#pragma unroll
                for (int k = 0; k < 16; ++k) {
                    const int q = (k0 + k) * 64 + lane;
                    if (q < full) {
                        const uint32_t e = uint32_t(q) * 4u;
                        const int r = int(div_f(e, a));
                        const int c = int(e) - r * a.n_features;
                        float *row = tile + r * RS;
                        const int s = swz<RS>(r);
                        row[(c + 0) ^ s] = v[k].x;
                        row[(c + 1) ^ s] = v[k].y;
                        row[(c + 2) ^ s] = v[k].z;
                        row[(c + 3) ^ s] = v[k].w;
                    }
                }
            }
            wave_sync();
            body(t);
        }
    } else {
        for (; t < a.n_tiles; t += stride) {
            wave_sync();
            stage_scalar<RS>(a, tile, t, lane);
            wave_sync();
            body(t);
        }
    }
}

// ---- data decomposition ---------------------------------------------------------------
template <int RS, bool VEC, bool TAB_LDS>
__global__ void __launch_bounds__(512) data_kernel(KArgs a) {
    extern __shared__ int4 lds[];
    const Slot *slots;
    const int32_t *exits;
    char *tiles = bind_tables<TAB_LDS>(a, lds, slots, exits);
    const int lane = threadIdx.x & 63;
    float *tile = reinterpret_cast<float *>(tiles) + (threadIdx.x >> 6) * (kTileRows * RS);
    const int D = a.depth;
    const int last = (1 << D) - 1;
    const float *my = tile + lane * RS;
    const int sw = swz<RS>(lane);

    tile_loop<RS, VEC>(a, tile, lane, [&](int64_t t) {
        int w = 0;
        int32_t code = -1;
        for (int level = 0; level < a.levels; ++level) {
            const int base = w << D;
            int h = 0;
            for (int k = 0; k < D; ++k) {
                const Slot s = slots[base + h];
                const float xv = my[s.f ^ sw];
                h = 2 * h + 1 + int(!(xv < s.t));
            }
            code = exits[base + h - last];
            if (code < 0) break;
            w = code;
        }
        store_out(a, t * kTileRows + lane, code);
    });
}

// ---- speculative decomposition --------------------------------------------------------
template <int RS, bool VEC, bool TAB_LDS, int D>
__global__ void __launch_bounds__(512) spec_kernel(KArgs a) {
    constexpr int S = 1 << D;          // lanes per record group
    using Bits = typename std::conditional<(S > 32), uint64_t, uint32_t>::type;
    extern __shared__ int4 lds[];
    const Slot *slots;
    const int32_t *exits;
    char *tiles = bind_tables<TAB_LDS>(a, lds, slots, exits);
    const int lane = threadIdx.x & 63;
    float *tile = reinterpret_cast<float *>(tiles) + (threadIdx.x >> 6) * (kTileRows * RS);
    const int seg = lane >> D;         // record group within the wavefront
    const int j = lane & (S - 1);      // slot (decision node) this lane evaluates
    const int seg_shift = seg * S;
    const Slot root = slots[j];        // window 0 is shared by every record

    // Evaluate one window level for the 64 records of the tile.  In round g, segment
    // `seg` evaluates record seg*S + g, so record r's outcome bits arrive in the segment
    // that lane r belongs to, in the round where g == r % S.
    auto eval_level = [&](bool first, int w) -> Bits {
        Bits bits = 0;
#pragma unroll 8
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
            const float xv = tile[r * RS + (p.f ^ swz<RS>(r))];
            const uint64_t m = __ballot(!(xv < p.t));
            if (j == g) bits = Bits(m >> seg_shift);
        }
        return bits;
    };
    auto walk = [&](Bits bits) -> int {
        int h = 0;
#pragma unroll
        for (int k = 0; k < D; ++k) h = 2 * h + 1 + int((bits >> h) & 1);
        return h - (S - 1);
    };

    tile_loop<RS, VEC>(a, tile, lane, [&](int64_t t) {
        int w = 0;
        int32_t code = exits[walk(eval_level(true, 0))];
        bool done = code < 0;
        if (!done) w = code;
        for (int level = 1; level < a.levels; ++level) {
            if (__all(done)) break;
            const Bits bits = eval_level(false, w);
            if (!done) {
                code = exits[(w << D) + walk(bits)];
                done = code < 0;
                if (!done) w = code;
            }
        }
        store_out(a, t * kTileRows + lane, code);
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
