// gfx950 forest kernel template, instantiated for int32 exit codes in forest.hip and for
// int16 ones in forest_ex16.hip (two translation units, compiled in parallel).
//
// Forests are evaluated tree after tree (the concatenated-trees scheme the paper cites
// in Section 1) and the trees' classes are combined by majority vote, ties going to the
// smallest class id.  Each record's votes live in registers as packed 8-bit counters.
//
// The tables of all trees together usually exceed the LDS, so a workgroup works on one
// group of tiles at a time (one 64-record tile per wavefront, staged once) and streams the
// trees' tables through the LDS in chunks of consecutive trees; every tree of a chunk is
// walked for the whole group before the next chunk replaces it.  All wavefronts of a
// workgroup iterate over the same groups and chunks, so the workgroup barriers around the
// chunk copies are reached uniformly.  Forests whose single trees do not fit the LDS read
// their tables from global memory instead.
#pragma once

#include "device_common.hpp"

namespace dtree {
namespace {

using dev::Slot;

// The tree and chunk descriptors never change during a launch and are read at wavefront-
// uniform indices: read them through the constant address space, which makes them scalar
// loads.  A vector load would share the in-order load counter with the record prefetch, so
// waiting for a descriptor would also wait for the next tile to arrive from HBM.
typedef int v4i __attribute__((ext_vector_type(4)));
typedef const __attribute__((address_space(4))) v4i ConstV4i;

__device__ __forceinline__ int4 read_const(const int4 *p, int i) {
    const v4i v = ((ConstV4i *)(p))[i];
    return int4{v.x, v.y, v.z, v.w};
}

typedef int v2i __attribute__((ext_vector_type(2)));
typedef const __attribute__((address_space(4))) v2i ConstV2i;

// Root slot of tree i's window 0 (from the per-tree root array): a scalar load that does
// not wait for the tree's descriptor.
__device__ __forceinline__ Slot read_root(const int2 *p, int i) {
    const v2i v = ((ConstV2i *)(p))[i];
    return Slot{__int_as_float(v.x), v.y};
}

template <int NV>
__device__ __forceinline__ void add_vote(uint32_t (&votes)[NV], int cls) {
    if constexpr (NV == 2) {
        // eight counters in one 64-bit word: a shift and a 64-bit add
        uint64_t v = uint64_t(votes[1]) << 32 | votes[0];
        v += uint64_t(1) << (cls * 8);
        votes[0] = uint32_t(v);
        votes[1] = uint32_t(v >> 32);
    } else {
        const int word = cls >> 2;
        const uint32_t inc = 1u << ((cls & 3) * 8);
#pragma unroll
        for (int r = 0; r < NV; ++r) votes[r] += (word == r) ? inc : 0u;
    }
}

// Class with the most votes; the strict comparison keeps the smallest id on ties.
template <int NV>
__device__ __forceinline__ int majority(const uint32_t (&votes)[NV], int n_classes) {
    int best = 0;
    int best_count = -1;
#pragma unroll
    for (int r = 0; r < NV; ++r) {
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            const int c = r * 4 + b;
            const int count = int((votes[r] >> (8 * b)) & 255u);
            if (c < n_classes && count > best_count) {
                best_count = count;
                best = c;
            }
        }
    }
    return best;
}

// Trees walked together per lane by the data decomposition.
constexpr int kIlp = 4;

// The whole chunk buffer, copied by the workgroup.
__device__ __forceinline__ void copy_chunk(const FArgs &a, int4 *tab, const int4 &ch) {
    const int4 *src = a.tables + (ch.z >> 4);
    for (int i = threadIdx.x; i < (ch.w >> 4); i += blockDim.x) tab[i] = src[i];
}

// Chunks of up to kStage * 16 bytes per thread are loaded into registers before the
// barrier that frees the chunk buffer, so the loads' latency overlaps the wait for the
// slowest wavefront; only the LDS writes sit between the two barriers.
constexpr int kStage = 2;

__device__ __forceinline__ void copy_chunk_staged(const FArgs &a, int4 *tab, const int4 &ch) {
    const v4i *src = reinterpret_cast<const v4i *>(a.tables) + (ch.z >> 4);
    v4i *dst = reinterpret_cast<v4i *>(tab);
    const int n16 = ch.w >> 4;                       // >= 1: a chunk holds a tree
    v4i v[kStage];
#pragma unroll
    for (int q = 0; q < kStage; ++q) {
        // unconditional loads (a thread past the end re-reads the last word): no branch
        // between the loads, so they are all in flight before the barrier
        const int i = int(threadIdx.x) + q * int(blockDim.x);
        v[q] = src[i < n16 ? i : n16 - 1];
    }
    __syncthreads();                                 // previous chunk no longer read
    // unconditional writes too (a thread past the end writes the last word again, the same
    // value its owner writes): with no branch around them, every load is waited for on one
    // path, and the compiler needs no catch-all wait later (which, the vector-memory counter
    // being in order, would also wait for the next record tiles' prefetch)
#pragma unroll
    for (int q = 0; q < kStage; ++q) {
        const int i = int(threadIdx.x) + q * int(blockDim.x);
        dst[i < n16 ? i : n16 - 1] = v[q];
    }
}

// SD = 0: data decomposition; SD > 0: speculative decomposition with window depth SD.
// EX: exit codes stored as int32, int16 where every code of the forest fits, or packed
// into the windows' bottom slots (dev::PackedExits) where every code fits 11 bits.
template <class EX, int RS, int LOAD, bool TAB_LDS, int NV, int SD>
__global__ void __launch_bounds__(64 * forest_max_waves(SD == 0 ? 0 : 1, SD, RS)) forest_kernel(FArgs a) {
    extern __shared__ int4 lds[];
    // compute-bound: wide rows unprefetched; the speculative walk with vector loads keeps
    // no prefetch either (its registers would not fit 16 wavefronts per CU)
    constexpr bool kPrefetch = LOAD != kLoadScalar && RS <= 32 && !(SD > 0 && LOAD == kLoadVec);
    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    float *tile = reinterpret_cast<float *>(lds) + wave * (kTileRows * RS);
    int4 *tab = lds + (a.waves * kTileRows * RS) / 4;   // chunk buffer after the tiles
    // The data decomposition reads each lane's own record: column-major tiles make every
    // such read conflict-free.  The speculative one reads across a record: row-major.
    constexpr int kLayout = SD == 0 ? dev::kColMajor : dev::kRowMajor;
    constexpr int kStride = SD == 0 ? kTileRows : 1;
    const float *row = SD == 0 ? tile + lane : tile + lane * RS;
    const int sw = SD == 0 ? 0 : dev::swz<RS>(lane);
    const int64_t n_groups = (a.in.n_tiles + a.waves - 1) / a.waves;

    // Speculative decomposition: exit code of this lane's record for the tree whose tables
    // start at `base` (int32 codes).
    auto eval_tree = [&](const char *base, int levels, int slot_bytes) -> int32_t {
        const Slot *sl = reinterpret_cast<const Slot *>(base);
        const int32_t *ex = reinterpret_cast<const int32_t *>(base + slot_bytes);
        using Spec = dev::Spec<kXF32, RS, SD == 0 ? 2 : SD>;
        static_assert(Spec::kLayout == dev::kRowMajor, "forest tiles are staged row-major");
        const Spec spec(lane);
        const Slot root = sl[spec.j];
        return spec.run(sl, ex, levels, root, tile);
    };

    // A forest whose tables form one chunk is copied once: the tables then stay for every
    // group.  Otherwise the chunks are copied in turn for each group.
    if constexpr (TAB_LDS) {
        if (a.n_chunks == 1) {
            copy_chunk(a, tab, read_const(a.chunks, 0));
            __syncthreads();
        }
    }
    const bool staged = a.table_lds_bytes <= kStage * 16 * int(blockDim.x);

    // Full tiles are prefetched one group ahead; the partial last tile is staged directly.
    const int64_t n_full = a.in.n / kTileRows;
    int64_t g = blockIdx.x;
    dev::VecTile<(kPrefetch ? RS : 4), LOAD == kLoadExact> buf;
    if constexpr (kPrefetch) {
        const int64_t t0 = g * a.waves + wave;
        if (g < n_groups && t0 < n_full) buf.load_full(a.in, t0, lane);
    }
    for (; g < n_groups; g += gridDim.x) {
        const int64_t t = g * a.waves + wave;
        const bool active = t < a.in.n_tiles;        // uniform per wavefront
        dev::wave_sync();
        if (active) {
            if (kPrefetch && t < n_full)
                buf.template store<kLayout>(a.in, tile, lane);
            else
                dev::stage_now<kXF32, RS, LOAD, kLayout>(a.in, tile, t, lane);
        }
        dev::wave_sync();
        // The next group's tiles are prefetched into registers: here, or, when the chunks
        // are copied for every group, after the last chunk's copy (its loads would
        // otherwise queue behind the prefetch on the in-order vector-memory counter, and the
        // first chunk copy would wait for the prefetch to arrive from HBM).
        const bool prefetch_late = TAB_LDS && a.n_chunks > 1;
        auto prefetch_next = [&]() {
            if constexpr (kPrefetch) {
                const int64_t tn = t + int64_t(gridDim.x) * a.waves;
                if (tn < n_full) buf.load_full(a.in, tn, lane);
            }
        };
        if (!prefetch_late) prefetch_next();

        uint32_t votes[NV];
#pragma unroll
        for (int r = 0; r < NV; ++r) votes[r] = 0u;
        for (int c = 0; c < a.n_chunks; ++c) {
            const int4 ch = read_const(a.chunks, c);             // {first, end, byte_off, bytes}
            if constexpr (TAB_LDS) {
                if (a.n_chunks > 1) {
                    if (staged) {
                        copy_chunk_staged(a, tab, ch);
                    } else {
                        __syncthreads();             // previous chunk no longer read
                        copy_chunk(a, tab, ch);
                    }
                    __syncthreads();
                    if (c == a.n_chunks - 1) prefetch_next();
                }
            }
            if (!active) continue;
            // tables of the chunk's trees: in the LDS chunk buffer (which starts at the
            // chunk's byte offset ch.z of the tables), or in place
            const char *cbase = TAB_LDS ? reinterpret_cast<const char *>(tab)
                                        : reinterpret_cast<const char *>(a.tables);
            const int cofs = TAB_LDS ? ch.z : 0;
            int k = ch.x;
            if constexpr (SD == 0) {
                // K trees of the chunk walked together from tree k0
                auto walk_group = [&](auto kk, int k0) {
                    constexpr int K = decltype(kk)::value;
                    const char *base[K];
                    Slot root[K];
                    int sb[K], lv[K];
                    int32_t code[K];
#pragma unroll
                    for (int i = 0; i < K; ++i) {
                        const int4 d = read_const(a.trees, k0 + i);   // {byte_off, slot_bytes, levels, 0}
                        root[i] = read_root(a.roots, k0 + i);
                        base[i] = cbase + (d.x - cofs);
                        sb[i] = d.y;
                        lv[i] = d.z;
                    }
                    // Both kinds of scalar loads complete here, before the walk: one wait
                    // for them all, instead of one for the roots and, after the root step,
                    // another for the descriptors (which the compiler would otherwise sink
                    // to their first use).
#pragma unroll
                    for (int i = 0; i < K; ++i)
                        asm volatile("" ::"s"(base[i]), "s"(sb[i]), "s"(lv[i]), "s"(root[i].t),
                                     "s"(root[i].f));
                    dev::walk_data_k<K, kStride, EX>(base, root, sb, lv, a.depth, row, sw, code);
#pragma unroll
                    for (int i = 0; i < K; ++i) add_vote(votes, ~code[i]);
                };
                for (; k + kIlp <= ch.y; k += kIlp) walk_group(std::integral_constant<int, kIlp>(), k);
                if (ch.y - k == 3)
                    walk_group(std::integral_constant<int, 3>(), k);
                else if (ch.y - k == 2)
                    walk_group(std::integral_constant<int, 2>(), k);
                else if (ch.y - k == 1)
                    walk_group(std::integral_constant<int, 1>(), k);
            } else {
                for (; k < ch.y; ++k) {
                    const int4 d = read_const(a.trees, k);   // {byte_off, slot_bytes, levels, 0}
                    add_vote(votes, ~eval_tree(cbase + (d.x - cofs), d.z, d.y));
                }
            }
        }
        if (active)
            dev::store_value(a.out, a.out_kind, a.in.n, t * kTileRows + lane,
                             majority(votes, a.n_classes));
    }
}

template <class EX, int RS, int LOAD, bool TAB_LDS, int NV>
const void *for_votes(int algo, int depth) {
    if (algo == kAlgoData)
        return reinterpret_cast<const void *>(&forest_kernel<EX, RS, LOAD, TAB_LDS, NV, 0>);
    if constexpr (std::is_same<EX, int32_t>::value) {   // narrower codes: data walk only
        if (depth == 2)
            return reinterpret_cast<const void *>(&forest_kernel<EX, RS, LOAD, TAB_LDS, NV, 2>);
        if (depth == 4)
            return reinterpret_cast<const void *>(&forest_kernel<EX, RS, LOAD, TAB_LDS, NV, 4>);
    }
    return nullptr;
}

template <class EX, int RS, int LOAD, bool TAB_LDS>
const void *for_tab(int algo, int vote_words, int depth) {
    switch (vote_words) {
        case 2: return for_votes<EX, RS, LOAD, TAB_LDS, 2>(algo, depth);
        case 4: return for_votes<EX, RS, LOAD, TAB_LDS, 4>(algo, depth);
        case 16: return for_votes<EX, RS, LOAD, TAB_LDS, 16>(algo, depth);
        default: return nullptr;
    }
}

template <class EX, int RS, int LOAD>
const void *for_load(int algo, bool tab_lds, int vote_words, int depth) {
    return tab_lds ? for_tab<EX, RS, LOAD, true>(algo, vote_words, depth)
                   : for_tab<EX, RS, LOAD, false>(algo, vote_words, depth);
}

template <class EX, int RS>
const void *for_stride(int algo, int load_mode, bool tab_lds, int vote_words, int depth) {
    switch (load_mode) {
        case kLoadScalar: return for_load<EX, RS, kLoadScalar>(algo, tab_lds, vote_words, depth);
        case kLoadVec: return for_load<EX, RS, kLoadVec>(algo, tab_lds, vote_words, depth);
        case kLoadExact: return for_load<EX, RS, kLoadExact>(algo, tab_lds, vote_words, depth);
        default: return nullptr;
    }
}

// Kernel instance for exit codes of type EX.
template <class EX>
const void *forest_kernel_for_ex(int algo, int row_stride, int load_mode, bool tables_in_lds,
                                 int vote_words, int depth) {
    switch (row_stride) {
        case 4: return for_stride<EX, 4>(algo, load_mode, tables_in_lds, vote_words, depth);
        case 8: return for_stride<EX, 8>(algo, load_mode, tables_in_lds, vote_words, depth);
        case 16: return for_stride<EX, 16>(algo, load_mode, tables_in_lds, vote_words, depth);
        case 32: return for_stride<EX, 32>(algo, load_mode, tables_in_lds, vote_words, depth);
        case 64: return for_stride<EX, 64>(algo, load_mode, tables_in_lds, vote_words, depth);
        case 128: return for_stride<EX, 128>(algo, load_mode, tables_in_lds, vote_words, depth);
        case 256: return for_stride<EX, 256>(algo, load_mode, tables_in_lds, vote_words, depth);
        default: return nullptr;
    }
}

}  // namespace
}  // namespace dtree
