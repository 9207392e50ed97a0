// Device building blocks shared by the single-tree and forest kernels (gfx950).
//
// Record tiles: every wavefront owns a private tile of 64 records (one per lane) in the
// LDS, in the records' own element type (fp32, fp16, bf16 or uint8).  Row r (record)
// starts at element r*RS; the 4-byte word w of a row is stored at word w ^ swz(r), bytes
// within a word unchanged.  The XOR spreads the 64 rows over all 64 banks for a fixed
// column, so the top levels of a tree (where every lane reads the same feature) are
// conflict-free, and the staging stores land on distinct banks.  Staging moves whole
// words and does not depend on the element type; a tree step widens the element it reads
// to fp32 (exactly) and compares it with the fp32 threshold.
//
// Window tables (built on the host, see encode.hpp): for window w, slot p in [1, 2^D)
// holds the (threshold, feature) of heap node p (children 2p, 2p+1; slot 0 is padding);
// exit e holds the next window (>= 0) or the result -(value + 1).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>
#include <utility>

#include "kernels.hpp"

namespace dtree {
namespace dev {

typedef float f32x4 __attribute__((ext_vector_type(4)));

struct alignas(8) Slot {
    float t;
    int32_t f;   // byte offset of the feature in an fp32 row: 4 * feature index
};

// The two children 2p, 2p+1 of a heap slot: one aligned 16-byte LDS read.
struct alignas(16) Slot2 {
    Slot l, r;
};

// Exit codes packed into the window's bottom slots (forest data walk): the 32-bit word of
// a slot p in [S/2, S) holds the feature's byte offset in bits 0-9 and the exit codes of
// its children 2p and 2p+1 (11-bit two's complement) in bits 10-20 and 21-31; slots
// above the bottom level hold the byte offset alone.  The exit is then known from the
// last slot of the window, with no read of an exit table.
struct PackedExits {};
constexpr int kPackedFeatureMask = 0x3FF;

// Word swizzle of row r for rows of RSW 4-byte words.
template <int RSW>
__device__ __forceinline__ int swz(int r) {
    if constexpr (RSW >= 64) {
        return r;                                  // r < 64 <= RSW
    } else {
        constexpr int sh = __builtin_ctz(64 / RSW);
        return (r >> sh) & (RSW - 1);
    }
}

// Record element types.  widen() is exact for every value (NaN stays NaN, fp16 and bf16
// subnormals become the same fp32 value), so a decision on a widened element is the
// decision on the value the element stores.
template <int XT> struct Elem;
template <> struct Elem<kXF32> {
    using T = float;
    static __device__ __forceinline__ float widen(float v) { return v; }
};
template <> struct Elem<kXF16> {
    using T = uint16_t;   // IEEE binary16 bits
    static __device__ __forceinline__ float widen(uint16_t b) {
        return float(__builtin_bit_cast(_Float16, b));
    }
};
template <> struct Elem<kXBF16> {
    using T = uint16_t;   // bfloat16 bits: the high half of an fp32
    static __device__ __forceinline__ float widen(uint16_t b) {
        return __uint_as_float(uint32_t(b) << 16);
    }
};
template <> struct Elem<kXU8> {
    using T = uint8_t;
    static __device__ __forceinline__ float widen(uint8_t b) { return float(b); }
};

// Window-table slots as the kernels for record type XT read them.
//   fp32 records: Slot {float t; int32 f} (8 bytes), decision !(x < t).
//   Narrow records: one 32-bit word, the feature index in the high half and in the low
//   half a key on the record type's grid (built on the host, see encode.hpp): for fp16 and
//   bf16 the threshold rounded up to the nearest value of the type, for uint8 its integer
//   ceiling clamped to 0..256.  No value of the type lies strictly between t and the key,
//   so !(x < key) on the stored element is the decision !(x < t) on its widened value.
template <int XT> struct Node;
template <> struct Node<kXF32> {
    using S = Slot;
    using Pair = Slot2;
    static __device__ __forceinline__ int feature(const Slot &s) { return s.f >> 2; }
    static __device__ __forceinline__ bool right(float x, const Slot &s) { return !(x < s.t); }
};
template <> struct Node<kXF16> {
    using S = uint32_t;
    struct alignas(8) Pair { uint32_t l, r; };
    static __device__ __forceinline__ int feature(uint32_t s) { return int(s >> 16); }
    static __device__ __forceinline__ bool right(uint16_t x, uint32_t s) {
        return !(Elem<kXF16>::widen(x) < Elem<kXF16>::widen(uint16_t(s)));
    }
};
template <> struct Node<kXBF16> {
    using S = uint32_t;
    struct alignas(8) Pair { uint32_t l, r; };
    static __device__ __forceinline__ int feature(uint32_t s) { return int(s >> 16); }
    static __device__ __forceinline__ bool right(uint16_t x, uint32_t s) {
        return !(Elem<kXBF16>::widen(x) < Elem<kXBF16>::widen(uint16_t(s)));
    }
};
template <> struct Node<kXU8> {
    using S = uint32_t;
    struct alignas(8) Pair { uint32_t l, r; };
    static __device__ __forceinline__ int feature(uint32_t s) { return int(s >> 16); }
    static __device__ __forceinline__ bool right(uint8_t x, uint32_t s) {
        return uint32_t(x) >= (s & 0xFFFFu);
    }
};

// Feature of slot `s` in a record row of the tile: element (feature ^ sw) * STRIDE of `row`.
// fp32 slots carry the feature as a byte offset, so the address is one xor-add.
template <int XT, int STRIDE>
__device__ __forceinline__ typename Elem<XT>::T feature_at(const typename Elem<XT>::T *row,
                                                           const typename Node<XT>::S &s, int sw) {
    if constexpr (XT == kXF32)
        return *reinterpret_cast<const float *>(reinterpret_cast<const char *>(row) +
                                                (s.f ^ (sw << 2)) * STRIDE);
    else
        return row[(Node<XT>::feature(s) ^ sw) * STRIDE];
}

// Element-level position swizzle for rows of RS elements of type XT: the word swizzle,
// scaled to elements (the position of an element within its word is unchanged).
template <int XT, int RS>
__device__ __forceinline__ int swz_el(int r) {
    constexpr int kPerWord = 4 / int(sizeof(typename Elem<XT>::T));
    return swz<RS / kPerWord>(r) * kPerWord;
}

// Ordering of LDS accesses among the lanes of one wavefront.  A wavefront's LDS
// instructions execute in order; the fences keep the compiler from moving accesses
// across this point.
__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ uint32_t div_f(uint32_t e, const Rows &in) {
    return in.n_features == 1 ? e : __umulhi(e, in.magic_f);
}

__device__ __forceinline__ uint32_t div_w(uint32_t e, const Rows &in) {
    return in.n_words == 1 ? e : __umulhi(e, in.magic_w);
}

// Records of tile `tile` (tiles of TR records) that exist in the input.
template <int TR = kTileRows>
__device__ __forceinline__ int valid_rows(const Rows &in, int64_t tile) {
    const int64_t left = in.n - tile * TR;
    return left < TR ? int(left) : TR;
}

// Tile layouts.  Row-major (the default): row r at word r*RSW, word w at w ^ swz(r).
// Column-major (fp32 only, used where every lane reads its own record): column c at word
// c*64, row r at c*64 + r, so lane r always reads bank r, whatever column it asks for.
// Flat row-major: row r at word r*RSW, word w at w, for kernels whose wavefront reads one
// row at a time (64-lane record groups): a single row is conflict-free without the
// swizzle, and staging then stores whole 16-byte vectors.
enum TileLayout { kRowMajor = 0, kColMajor = 1, kRowFlat = 2 };

// Store 4 consecutive words (c % 4 == 0) of row r into the tile (rows of RSW words;
// `tile` is the word view of the tile).
template <int RSW, int LAYOUT = kRowMajor>
__device__ __forceinline__ void put4(float *tile, int r, int c, f32x4 v) {
    if constexpr (LAYOUT == kColMajor) {   // 64-record tiles only
        tile[(c + 0) * kTileRows + r] = v.x;
        tile[(c + 1) * kTileRows + r] = v.y;
        tile[(c + 2) * kTileRows + r] = v.z;
        tile[(c + 3) * kTileRows + r] = v.w;
        return;
    }
    if constexpr (LAYOUT == kRowFlat) {
        *reinterpret_cast<f32x4 *>(tile + r * RSW + c) = v;
        return;
    }
    float *row = tile + r * RSW;
    const int s = swz<RSW>(r);
    row[(c + 0) ^ s] = v.x;
    row[(c + 1) ^ s] = v.y;
    row[(c + 2) ^ s] = v.z;
    row[(c + 3) ^ s] = v.w;
}

// Vectorised staging (dense rows of n_words 4-byte words, n_words % 4 == 0, 16-byte
// aligned base), one tile of TR records held in registers so that the next tile's loads
// overlap the walk of the current one.  RSW = LDS row stride in words.  The element type
// does not matter here: words are moved unchanged.
//
// Loads are never guarded by a branch: guarded loads compile into branches whose joins
// copy the loaded registers, which forces a wait for every outstanding load right after
// the prefetch is issued.  A lane whose vector lies past the tile's valid data re-reads
// the last valid vector instead, so rows past the end of the input hold copies of valid
// features; their results are never stored.  EXACT (n_words == RSW): every lane owns
// RSW/4 vectors of a full tile and the LDS positions are shifts and masks.
template <int RSW, bool EXACT, int TR = kTileRows>
struct VecTile {
    static constexpr int kVec = TR * RSW / 256;   // 16-byte vectors per lane for n_words == RSW
    static_assert(kVec >= 1, "vector staging needs one 16-byte vector per lane and tile");
    f32x4 v[kVec];

    __device__ __forceinline__ const f32x4 *base(const Rows &in, int64_t tile) const {
        return reinterpret_cast<const f32x4 *>(static_cast<const char *>(in.x) +
                                               tile * TR * in.n_words * 4);
    }

    // Any tile; nvec = vectors holding valid records (>= 1).
    __device__ __forceinline__ void load_clamped(const Rows &in, int64_t tile, int lane, int nvec) {
        const f32x4 *src = base(in, tile);
#pragma unroll
        for (int k = 0; k < kVec; ++k) {
            const int q = k * 64 + lane;
            v[k] = __builtin_nontemporal_load(src + (q < nvec ? q : nvec - 1));
        }
    }

    // Tile with 64 valid records.
    __device__ __forceinline__ void load_full(const Rows &in, int64_t tile, int lane) {
        if constexpr (EXACT) {
            const f32x4 *src = base(in, tile) + lane;
#pragma unroll
            for (int k = 0; k < kVec; ++k) v[k] = __builtin_nontemporal_load(src + k * 64);
        } else {
            load_clamped(in, tile, lane, TR * in.n_words / 4);
        }
    }

    __device__ __forceinline__ void store_col_major(float *tile, int lane) const;

    // Any tile, including the partial last one.
    __device__ __forceinline__ void load_tail(const Rows &in, int64_t tile, int lane) {
        load_clamped(in, tile, lane, (valid_rows<TR>(in, tile) * in.n_words) >> 2);
    }

    template <int LAYOUT = kRowMajor>
    __device__ __forceinline__ void store(const Rows &in, float *tile, int lane) const {
        if constexpr (EXACT && LAYOUT == kColMajor && RSW <= 32) {
            // (wider rows keep the plain stores: the butterfly's 2 x RSW registers would
            // not fit the forest kernel's 128)
            store_col_major(tile, lane);
        } else if constexpr (EXACT) {
            constexpr int sh = __builtin_ctz(RSW);
#pragma unroll
            for (int k = 0; k < kVec; ++k) {
                const int e = (k * 64 + lane) * 4;
                put4<RSW, LAYOUT>(tile, e >> sh, e & (RSW - 1), v[k]);
            }
        } else {
            const int full = TR * in.n_words / 4;
#pragma unroll
            for (int k = 0; k < kVec; ++k) {
                const int q = k * 64 + lane;
                if (q < full) {
                    const uint32_t e = uint32_t(q) * 4u;
                    const int r = int(div_w(e, in));
                    put4<RSW, LAYOUT>(tile, r, int(e) - r * in.n_words, v[k]);
                }
            }
        }
    }
};

// Column-major stores of a full exact tile without bank conflicts (64-record tiles).  With
// L = RSW / 4 lanes per row, lane l = a*L + b holds in v[k] the words 4b..4b+3 of row
// k*(64/L) + a.  Storing one register at a time would send 64 lanes to only 64/L rows,
// i.e. 64/L banks of a column-major tile (an L-way conflict).  Store j instead takes
// v[b ^ j] in every lane: its rows (b ^ j)*(64/L) + a are 64 distinct rows, so each store
// touches every bank once.  The per-lane choice of register is an XOR butterfly of selects
// (log2 L stages of conditional swaps), after which w[j] == v[b ^ j].
template <int RSW, bool EXACT, int TR>
__device__ __forceinline__ void store_col_major_tile(const f32x4 (&v)[RSW / 4], float *tile, int lane) {
    constexpr int L = RSW / 4;                  // lanes per row = vectors per lane
    constexpr int R = 64 / L;                   // rows per load instruction
    static_assert(TR == kTileRows && L >= 1 && (L & (L - 1)) == 0, "64-record exact tiles");
    const int a = lane / L, b = lane % L;
    f32x4 w[L];
#pragma unroll
    for (int k = 0; k < L; ++k) w[k] = v[k];
#pragma unroll
    for (int bit = 1; bit < L; bit <<= 1) {
        const bool swap = (b & bit) != 0;
#pragma unroll
        for (int k = 0; k < L; ++k) {
            if (k & bit) continue;
            const f32x4 lo = w[k], hi = w[k | bit];
            w[k] = swap ? hi : lo;
            w[k | bit] = swap ? lo : hi;
        }
    }
    // word (4b + i)*64 + (b ^ j)*R + a of the tile
    float *col = tile + (4 * b) * kTileRows + a;
#pragma unroll
    for (int j = 0; j < L; ++j) {
        float *dst = col + (b ^ j) * R;
        dst[0 * kTileRows] = w[j].x;
        dst[1 * kTileRows] = w[j].y;
        dst[2 * kTileRows] = w[j].z;
        dst[3 * kTileRows] = w[j].w;
    }
}

template <int RSW, bool EXACT, int TR>
__device__ __forceinline__ void VecTile<RSW, EXACT, TR>::store_col_major(float *tile, int lane) const {
    store_col_major_tile<RSW, EXACT, TR>(v, tile, lane);
}

// Vectorised staging of wide rows (RSW > 64 words) in chunks of 16 vectors per lane,
// without prefetch (loads clamped to the valid vectors as in VecTile).
template <int RSW, int LAYOUT = kRowMajor, int TR = kTileRows>
__device__ __forceinline__ void stage_wide(const Rows &in, float *tile, int64_t t, int lane) {
    const int nvec = (valid_rows<TR>(in, t) * in.n_words) >> 2;
    const int full = TR * in.n_words / 4;
    const f32x4 *src = reinterpret_cast<const f32x4 *>(static_cast<const char *>(in.x) +
                                                       t * TR * in.n_words * 4);
#pragma unroll 1
    for (int k0 = 0; k0 < TR * RSW / 256; k0 += 16) {
        f32x4 v[16];
#pragma unroll
        for (int k = 0; k < 16; ++k) {
            const int q = (k0 + k) * 64 + lane;
            v[k] = __builtin_nontemporal_load(src + (q < nvec ? q : nvec - 1));
        }
#pragma unroll
        for (int k = 0; k < 16; ++k) {
            const int q = (k0 + k) * 64 + lane;
            if (q < full) {
                const uint32_t e = uint32_t(q) * 4u;
                const int r = int(div_w(e, in));
                put4<RSW, LAYOUT>(tile, r, int(e) - r * in.n_words, v[k]);
            }
        }
    }
}

// General staging: any ld >= F, element-aligned, one element per load.
template <int XT, int RS, int LAYOUT = kRowMajor, int TR = kTileRows>
__device__ __forceinline__ void stage_scalar(const Rows &in, float *tile_words, int64_t t,
                                             int lane) {
    static_assert(LAYOUT != kColMajor || XT == kXF32, "column-major tiles hold fp32 records");
    using T = typename Elem<XT>::T;
    T *tile = reinterpret_cast<T *>(tile_words);
    const T *x = static_cast<const T *>(in.x);
    static_assert(LAYOUT != kColMajor || TR == kTileRows, "column-major tiles hold 64 records");
    const int64_t row0 = t * TR;
    const int valid = valid_rows<TR>(in, t);
    // TR * F elements, 64 per pass (TR is 32 or 64)
    for (int k = 0; k < (TR == kTileRows ? in.n_features : (in.n_features + 1) >> 1); ++k) {
        const uint32_t idx = uint32_t(k * 64 + lane);
        const int r = int(div_f(idx, in));
        const int c = int(idx) - r * in.n_features;
        if (r >= TR) break;            // only in the last pass of a 32-record tile, odd F
        T v = T(0);
        if (r < valid) v = x[(row0 + r) * in.ld + c];
        if constexpr (LAYOUT == kColMajor)
            tile[c * kTileRows + r] = v;
        else if constexpr (LAYOUT == kRowFlat)
            tile[r * RS + c] = v;
        else
            tile[r * RS + (c ^ swz_el<XT, RS>(r))] = v;
    }
}

// LDS row stride in words of a row of RS elements of XT, and whether the vector staging
// path (16-byte loads, at least one vector per lane and row) exists for it.
template <int XT, int RS>
constexpr int row_words() { return RS * int(sizeof(typename Elem<XT>::T)) / 4; }
template <int XT, int RS, int TR = kTileRows>
constexpr bool has_vec_staging() { return TR * row_words<XT, RS>() >= 256; }

// Stage tile t (of TR records) without register prefetch.
template <int XT, int RS, int LOAD, int LAYOUT = kRowMajor, int TR = kTileRows>
__device__ __forceinline__ void stage_now(const Rows &in, float *tile, int64_t t, int lane) {
    constexpr int RSW = row_words<XT, RS>();
    if constexpr (LOAD != kLoadScalar && has_vec_staging<XT, RS, TR>() && RSW <= 64) {
        VecTile<RSW, LOAD == kLoadExact, TR> buf;
        buf.load_tail(in, t, lane);
        buf.template store<LAYOUT>(in, tile, lane);
    } else if constexpr (LOAD != kLoadScalar && has_vec_staging<XT, RS, TR>()) {
        stage_wide<RSW, LAYOUT, TR>(in, tile, t, lane);
    } else {
        stage_scalar<XT, RS, LAYOUT, TR>(in, tile, t, lane);
    }
}

// v_writelane_b32: `value` (wavefront-uniform) written into lane `lane` of `old`.  The
// compiler's intrinsic has no clang builtin here, so it is declared by its LLVM name.
extern "C" __device__ int dt_llvm_writelane(int value, int lane, int old)
    __asm("llvm.amdgcn.writelane.i32");

__device__ __forceinline__ uint32_t writelane(uint32_t value, int lane, uint32_t old) {
    return uint32_t(dt_llvm_writelane(int(value), lane, int(old)));
}

// One heap step, p <- 2p + b, as a single add with carry: the compare that produces b
// leaves it as a wave mask in scalar registers, which v_addc takes as its carry-in, so
// the step costs one vector instruction instead of a select and a shift-or.  Lanes
// outside the active mask are not written.
__device__ __forceinline__ int heap_step(int p, bool b) {
    const uint64_t m = __ballot(b);
    int q;
    uint64_t carry_out;
    asm("v_addc_co_u32_e64 %0, %1, %2, %2, %3" : "=v"(q), "=s"(carry_out) : "v"(p), "s"(m));
    return q;
}

// ---- data decomposition: the record of this lane walks one tree --------------------------
// Within a window the record descends p <- 2p + !(x[f_p] < t_p) for exactly D steps
// (Procedure 2's "child + predicate" step on the 1-based heap), then the exit names the next
// window or the result.  One-level lookahead: while node p's feature is read, both children
// of p are fetched as one 16-byte pair and the comparison selects between them, so each
// level costs one LDS round trip instead of two dependent ones.
// `row[(f ^ sw) * STRIDE]` is feature f of this lane's record: STRIDE 1 for row-major
// tiles, kTileRows (and sw = 0) for column-major ones.  Exit codes are EX: int32, or int16
// where a forest's codes all fit (sign-extended when read).
// `root0` is slot 1 of window 0, the same for every record (read once by the caller).
// The bottom step reads the exits of both children of its node together with the node's
// feature, and the comparison picks one: no exit read after the last comparison.
template <int XT, int STRIDE = 1, class EX = int32_t>
__device__ __forceinline__ int32_t walk_data(const typename Node<XT>::S *slots,
                                             const EX *exits, int D, int levels,
                                             const typename Elem<XT>::T *row, int sw,
                                             const typename Node<XT>::S &root0) {
    using N = Node<XT>;
    using NS = typename N::S;
    using Pair = typename N::Pair;
    struct alignas(2 * sizeof(EX)) ExitPair { EX l, r; };
    const int S = 1 << D;
    int w = 0;
    int32_t code = -1;
    for (int level = 0; level < levels; ++level) {
        const NS *win = slots + (w << D);
        int p = 1;
        NS s = level == 0 ? root0 : win[1];
        for (int k = 1; k < D; ++k) {
            const auto xv = feature_at<XT, STRIDE>(row, s, sw);
            const Pair kids = *reinterpret_cast<const Pair *>(win + 2 * p);
            const bool right = N::right(xv, s);
            p = heap_step(p, right);
            s = right ? kids.r : kids.l;
        }
        // exits of children 2p and 2p + 1 of the bottom node p: an aligned pair (2p - S is
        // even)
        const ExitPair e = *reinterpret_cast<const ExitPair *>(exits + (w << D) + 2 * p - S);
        const auto xv = feature_at<XT, STRIDE>(row, s, sw);
        code = int32_t(N::right(xv, s) ? e.r : e.l);
        if (code < 0) break;
        w = code;
    }
    return code;
}

// Data decomposition over K trees at once (forests): the K walks of one record are
// independent, so interleaving them keeps K LDS dependency chains in flight per lane.
// Tree i's tables start at base[i] (LDS or global memory) and its window 0's root slot
// (slot 1) is root[i], a wavefront-uniform value; all trees share the window depth D.
template <int K, int STRIDE = 1, class EX = int32_t>
__device__ __forceinline__ void walk_data_k(const char *const (&base)[K],
                                            const Slot (&root)[K],
                                            const int (&slot_bytes)[K], const int (&levels)[K],
                                            int D, const float *row, int sw, int32_t (&code)[K]) {
    // K independent chains already hide the LDS latency, so each level reads just the
    // node's own 8-byte slot (no lookahead): fewer LDS bytes and bank conflicts per step.
    const int S = 1 << D;
    int w[K], p[K];
    int max_levels = 0;
#pragma unroll
    for (int i = 0; i < K; ++i) {
        w[i] = 0;
        p[i] = 1;
        code[i] = 0;
        max_levels = levels[i] > max_levels ? levels[i] : max_levels;
    }
    // Every walk starts at the root of window 0, whose slot is the same for every lane: it
    // comes from scalar registers, which saves one LDS slot read per tree (the LDS pipe is
    // one of this walk's bounds).  The next level's two slots are cheaper to read from the
    // LDS (two addresses: no bank conflicts) than to select from scalars (measured: four
    // vector instructions more per tree, 419 against 408 us on a 32-tree forest).  With
    // packed exits the window's bottom level always comes from the LDS (its slots carry the
    // exits).
    constexpr bool kPacked = std::is_same<EX, PackedExits>::value;
    int k0 = 0;
    if (D >= (kPacked ? 2 : 1)) {
        // the K feature reads first, then the K steps: one wait for all of them
        float xv[K];
#pragma unroll
        for (int i = 0; i < K; ++i) xv[i] = feature_at<kXF32, STRIDE>(row, root[i], sw);
#pragma unroll
        for (int i = 0; i < K; ++i) p[i] = heap_step(1, !(xv[i] < root[i].t));
        k0 = 1;
    }
    for (int level = 0; level < max_levels; ++level) {
        const Slot *win[K];
#pragma unroll
        for (int i = 0; i < K; ++i) win[i] = reinterpret_cast<const Slot *>(base[i]) + (w[i] << D);
        for (int k = level == 0 ? k0 : 0; k < (kPacked ? D - 1 : D); ++k) {
#pragma unroll
            for (int i = 0; i < K; ++i) {
                const Slot s = win[i][p[i]];
                const float xv = feature_at<kXF32, STRIDE>(row, s, sw);
                p[i] = heap_step(p[i], !(xv < s.t));
            }
        }
        // Every chain takes its exit, finished or not (a finished chain re-walked its last
        // window, so the index stays inside that window's exits), the K reads issued
        // together; a chain still running at this level has level < levels[i].
        int32_t c[K];
        if constexpr (kPacked) {
            // the bottom step: the slot's word names the feature and both exits (the 11-bit
            // field at bit 10 or bit 21, sign-extended)
#pragma unroll
            for (int i = 0; i < K; ++i) {
                const Slot s = win[i][p[i]];
                const Slot node{s.t, int(__builtin_amdgcn_ubfe(uint32_t(s.f), 0, 10))};
                const float xv = feature_at<kXF32, STRIDE>(row, node, sw);
                c[i] = __builtin_amdgcn_sbfe(s.f, !(xv < s.t) ? 21u : 10u, 11u);
            }
        } else {
#pragma unroll
            for (int i = 0; i < K; ++i)
                c[i] = int32_t(reinterpret_cast<const EX *>(base[i] + slot_bytes[i])[(w[i] << D) + p[i] - S]);
        }
        if (max_levels == 1) {            // one window per tree: the exits are the results
#pragma unroll
            for (int i = 0; i < K; ++i) code[i] = c[i];
            break;
        }
        bool all_done = true;
#pragma unroll
        for (int i = 0; i < K; ++i) {
            const bool live = code[i] >= 0;
            w[i] = live && c[i] >= 0 ? c[i] : w[i];
            code[i] = live ? c[i] : code[i];
            all_done = all_done && code[i] < 0;
            p[i] = 1;
        }
        if (__all(all_done)) break;
    }
}

// ---- speculative decomposition: a tile of 64 records through one tree -------------------
// A segment of S = 2^D lanes is the record group of one record: lane j evaluates heap slot
// j of the record's current window (the processor-node map of Procedure 5), so one
// wavefront instruction evaluates 64/S records' windows.  One ballot gathers the 64
// outcomes; record r's segment is handed to lane r, which walks its bits from the window
// root to the exit.
template <int XT, int RS, int D, int TR = kTileRows>
struct Spec {
    using T = typename Elem<XT>::T;
    using N = Node<XT>;
    using Slot = typename N::S;
    static constexpr int S = 1 << D;
    // Tiles of TR records: 64, or 32 for 32- and 64-lane groups.  A round evaluates one
    // record per group, so kRounds = TR S / 64 rounds cover the tile: group s evaluates
    // records s kRounds .. s kRounds + kRounds - 1, and record s kRounds + g lives in lane
    // s S + g (its group's lane g).  Only 32-record tiles of 32-lane groups leave lanes
    // without a record (g >= 16); in_record_order() moves the results to lanes 0 .. TR - 1.
    static_assert(TR == kTileRows || (S >= 32 && TR == 32), "32-record tiles need 32- or 64-lane groups");
    static constexpr int kRounds = TR * S / kTileRows;
    using Bits = typename std::conditional<(S > 32), uint64_t, uint32_t>::type;
    int j;          // slot evaluated by this lane (slot 0 is padding)
    int seg_shift;  // first lane of this lane's segment
    int rec_base;   // first record of this lane's segment (segment index * kRounds)

    // Record tile layout the rounds read.  64- and 32-lane groups read one or two record
    // rows per round: flat rows, so that a round's row is its group's first row plus a
    // constant (an instruction offset; a per-row swizzle would be a per-round register).
    // Narrower groups read 64/S rows at once, and the swizzle keeps rows reading the same
    // feature on distinct banks.
    static constexpr int kLayout = S >= 32 ? kRowFlat : kRowMajor;

    __device__ __forceinline__ explicit Spec(int lane)
        : j(lane & (S - 1)), seg_shift(lane & ~(S - 1)), rec_base((lane >> D) * kRounds) {}

    // Value wb of lane seg_shift + G (record seg_shift + G's window byte offset) in every
    // lane of the segment, with the round index G a compile-time constant:
    //   2, 4, 16 lanes: one DPP move (quad_perm within groups of 4 lanes, row_share within
    //     rows of 16), which folds into the slot address add;
    //   8, 32 lanes: ds_swizzle in bitmask mode (within each half-wave, lane i reads lane
    //     (i & and_mask) | G): no address computation, no VALU instruction;
    //   64 lanes: readlane into a scalar register.
    // Every source lane is in range and enabled, so no old value is needed.
    template <int G>
    __device__ __forceinline__ int window_of(int wb) const {
        if constexpr (S == 64)
            return __builtin_amdgcn_readlane(wb, G);
        else if constexpr (S == 32)
            return __builtin_amdgcn_ds_swizzle(wb, G << 5);          // and 0, or G
        else if constexpr (S == 16)
            return __builtin_amdgcn_mov_dpp(wb, 0x150 + G, 0xF, 0xF, true);   // row_share
        else if constexpr (S == 8)
            return __builtin_amdgcn_ds_swizzle(wb, G << 5 | 0x18);   // and 0b11000, or G
        else if constexpr (S == 4)
            return __builtin_amdgcn_mov_dpp(wb, G * 0x55, 0xF, 0xF, true);    // quad_perm
        else   // S == 2: quad_perm [G, G, 2 + G, 2 + G]
            return __builtin_amdgcn_mov_dpp(wb, G | G << 2 | (2 + G) << 4 | (2 + G) << 6,
                                            0xF, 0xF, true);
    }

    // Round G's mask m (bit i: slot i - seg_shift of record seg_shift + G, for the lanes i
    // of each segment) goes to lane seg_shift + G as that record's bits.  Segments of 32 and
    // 64 lanes write the scalar mask straight into the lane (v_writelane: one instruction
    // per 32 bits); narrower ones shift the mask by the segment and select the lane.
    template <int G>
    __device__ __forceinline__ void take(Bits &bits, uint64_t m) const {
        if constexpr (S == 64) {
            const uint32_t lo = writelane(uint32_t(m), G, uint32_t(bits));
            const uint32_t hi = writelane(uint32_t(m >> 32), G, uint32_t(bits >> 32));
            bits = uint64_t(hi) << 32 | lo;
        } else if constexpr (S == 32) {
            bits = writelane(uint32_t(m), G, bits);
            bits = writelane(uint32_t(m >> 32), 32 + G, bits);
        } else {
            if (j == G) bits = Bits(m >> seg_shift);
        }
    }

    // Rounds G0 + G... as one batch: the slot reads of every round are issued, then the
    // feature reads, then the compares, so a batch waits for two LDS round trips rather
    // than two per round.  In round g the segment starting at lane b evaluates record
    // b + g, so record r's bits arrive in r's own lane in the round g == r % S.  A
    // scheduling barrier after each batch keeps the compiler from holding every round's
    // loads in registers at once.
    template <int G0, int... G>
    __device__ __forceinline__ void eval_batch(std::integer_sequence<int, G...>, Bits &bits,
                                               const Slot *slots, bool first, const Slot &root,
                                               int wb, const T *tile) const {
        constexpr int K = sizeof...(G);
        Slot p[K];
        // wb: byte offset of the record's window, window id * 2^D * sizeof(Slot); added to
        // this lane's own slot address
        ((p[G] = first ? root
                       : *reinterpret_cast<const Slot *>(
                             reinterpret_cast<const char *>(slots + j) + window_of<G0 + G>(wb))),
         ...);
        T xv[K];
        ((xv[G] = feature_at<XT, 1>(tile + (rec_base + G0 + G) * RS, p[G],
                                    kLayout == kRowFlat ? 0 : swz_el<XT, RS>(rec_base + G0 + G))),
         ...);
        (take<G0 + G>(bits, __ballot(N::right(xv[G], p[G]))), ...);
        __builtin_amdgcn_sched_barrier(0);
    }

    template <int K, int... Q>
    __device__ __forceinline__ void eval_batches(std::integer_sequence<int, Q...>,
                                                 std::integral_constant<int, K>, Bits &bits,
                                                 const Slot *slots, bool first, const Slot &root,
                                                 int wb, const T *tile) const {
        (eval_batch<Q * K>(std::make_integer_sequence<int, K>(), bits, slots, first, root, wb,
                           tile),
         ...);
    }

    // Rounds per batch: 8, or 4 where the tile's prefetch buffer takes 64 registers (16 KiB
    // record tiles), which leaves too few for eight rounds' loads; never more than a level's
    // rounds.
    static constexpr int kPrefetchRegs = TR * RS * int(sizeof(T)) / 256;
    static constexpr int kMaxBatch = kPrefetchRegs >= 64 ? 4 : 8;
    static constexpr int kBatch = kRounds < kMaxBatch ? kRounds : kMaxBatch;
    static_assert(kBatch >= 1 && kRounds % kBatch == 0, "batches must cover a level's rounds");

    // One window level for the tile's records.
    __device__ __forceinline__ Bits eval(const Slot *slots, bool first, const Slot &root, int w,
                                         const T *tile) const {
        Bits bits = 0;
        eval_batches(std::make_integer_sequence<int, kRounds / kBatch>(),
                     std::integral_constant<int, kBatch>(), bits, slots, first, root,
                     first ? 0 : w * int(sizeof(Slot) << D), tile);
        return bits;
    }

    // Exit index reached from the window root (slot 1) by following the bits: p <- 2p + b_p.
    __device__ __forceinline__ int walk(Bits bits) const {
        int p = 1;
#pragma unroll
        for (int k = 0; k < D; ++k) p = 2 * p + int((bits >> p) & 1);
        return p - S;
    }

    // Windows of 2 or 4 slots have all their exits in one 8- or 16-byte word: a lane
    // reads its record's exits together with the slot reads of the level, so the exit is
    // picked from registers once the bits are walked instead of read after the walk.
    static constexpr bool kExitWord = S == 2 || S == 4;
    typedef int32_t ExitWord __attribute__((ext_vector_type(S == 4 ? 4 : 2)));

    static __device__ __forceinline__ int32_t pick(const ExitWord &e, int i) {
        if constexpr (S == 4) {
            const int32_t lo = (i & 1) ? e.y : e.x;
            const int32_t hi = (i & 1) ? e.w : e.z;
            return (i & 2) ? hi : lo;
        } else {
            return (i & 1) ? e.y : e.x;
        }
    }

    // Exit code of every lane's record.  `root` = slots[j] of window 0.  All 64 lanes
    // must be active.
    __device__ __forceinline__ int32_t run(const Slot *slots, const int32_t *exits, int levels,
                                           const Slot &root, const T *tile) const {
        if constexpr (kExitWord) {
            using EW = ExitWord;
            const EW *ew = reinterpret_cast<const EW *>(exits);
            int w = 0;
            const EW e0 = ew[0];
            int32_t code = pick(e0, walk(eval(slots, true, root, 0, tile)));
            bool done = code < 0;
            if (!done) w = code;
            for (int level = 1; level < levels; ++level) {
                if (__all(done)) break;
                const EW e = ew[w];             // w stays a valid window once done
                const Bits bits = eval(slots, false, root, w, tile);
                if (!done) {
                    code = pick(e, walk(bits));
                    done = code < 0;
                    if (!done) w = code;
                }
            }
            return code;
        } else {
            int w = 0;
            int32_t code = exits[walk(eval(slots, true, root, 0, tile))];
            bool done = code < 0 || (TR < kTileRows && j >= kRounds);   // lanes without a record
            if (!done) w = code;
            for (int level = 1; level < levels; ++level) {
                if (__all(done)) break;
                const Bits bits = eval(slots, false, root, w, tile);
                if (!done) {
                    code = exits[(w << D) + walk(bits)];
                    done = code < 0;
                    if (!done) w = code;
                }
            }
            return code;
        }
    }

    // Lane r's result for record r of the tile (r < TR).  With 32-record tiles of 32-lane
    // groups, records 16..31 live in lanes 32..47: one ds_bpermute brings them down.
    __device__ __forceinline__ int32_t in_record_order(int32_t v) const {
        if constexpr (S == 32 && TR == 32) {
            const int lane = seg_shift + j;
            const int src = lane < 16 ? lane : lane + 16;   // lanes >= 32 carry no record
            return __builtin_amdgcn_ds_bpermute((src & 63) << 2, v);
        } else {
            return v;
        }
    }
};

// Cooperative copy of n16 16-byte words from global memory into the LDS by the whole
// workgroup, eight loads in flight per thread (a plain loop would wait for each load's
// round trip before issuing the next).
__device__ __forceinline__ void copy_to_lds(int4 *dst, const int4 *src, int n16) {
    const int step = int(blockDim.x);
    int i = int(threadIdx.x);
    for (; i + 7 * step < n16; i += 8 * step) {
        int4 v[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) v[k] = src[i + k * step];
#pragma unroll
        for (int k = 0; k < 8; ++k) dst[i + k * step] = v[k];
    }
    for (; i < n16; i += step) dst[i] = src[i];
}

// ---- single-tree kernel scaffolding ------------------------------------------------------

// Window tables: staged into the LDS once per workgroup (TAB_LDS), or read in place from
// global memory.  Returns the first LDS byte after the tables (where record tiles start).
template <bool TAB_LDS, class NS>
__device__ __forceinline__ char *bind_tables(const KArgs &a, int4 *lds, const NS *&slots,
                                             const int32_t *&exits) {
    if constexpr (TAB_LDS) {
        const int ns = a.slot_bytes >> 4;
        const int ne = a.exit_bytes >> 4;
        copy_to_lds(lds, a.slots, ns);
        copy_to_lds(lds + ns, a.exits, ne);
        __syncthreads();
        slots = reinterpret_cast<const NS *>(lds);
        exits = reinterpret_cast<const int32_t *>(reinterpret_cast<const char *>(lds) + a.slot_bytes);
        return reinterpret_cast<char *>(lds) + a.slot_bytes + a.exit_bytes;
    } else {
        slots = reinterpret_cast<const NS *>(a.slots);
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
    if (a.out_vec) {   // dst is 16-byte aligned: r0 is a multiple of 32 or 64 records
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

// Persistent tile loop over tiles of TR records.  Wavefront g of G takes the contiguous
// tile range [g*chunk, (g+1)*chunk), chunk = ceil(tiles / G), so its results form one
// contiguous run of the output.  `body(t)` walks staged tile t and returns each lane's
// result (lane r: record r of the tile; lanes >= TR have none).  No workgroup barrier
// inside: the wavefronts of a workgroup process different numbers of tiles.
template <int XT, int RS, int LOAD, int LAYOUT = kRowMajor, int TR = kTileRows, class Body>
__device__ __forceinline__ void tile_loop(const KArgs &a, float *tile, uint8_t *obuf, int lane,
                                          Body body) {
    constexpr int RSW = row_words<XT, RS>();
    const int64_t G = int64_t(gridDim.x) * a.waves;
    const int64_t gw = int64_t(blockIdx.x) * a.waves + (threadIdx.x >> 6);
    const int64_t chunk = (a.in.n_tiles + G - 1) / G;
    const int64_t t0 = gw * chunk < a.in.n_tiles ? gw * chunk : a.in.n_tiles;
    const int64_t t1 = t0 + chunk < a.in.n_tiles ? t0 + chunk : a.in.n_tiles;
    const int64_t n_full = a.in.n / TR;            // tiles with TR valid records
    const int esize = a.out_kind == 0 ? 1 : 4;
    int64_t fl = t0;                               // first tile whose results are buffered

    auto finish = [&](int64_t t, int32_t v) {
        const int slot = int(t - fl) * TR + lane;
        if (TR == kTileRows || lane < TR) {
            if (esize == 1)
                obuf[slot] = uint8_t(v);
            else
                reinterpret_cast<int32_t *>(obuf)[slot] = v;
        }
        if (t - fl == a.out_cap - 1 || t + 1 == t1) {
            wave_sync();
            flush_results(a, obuf, fl * TR, (t + 1) * TR, lane);
            wave_sync();
            fl = t + 1;
        }
    };

    if constexpr (LOAD != kLoadScalar && has_vec_staging<XT, RS, TR>() && RSW <= 64) {
        // Full tiles: the loads of tile t + 1 are in flight in registers while tile t is
        // walked.  The partial last tile of the input, if any, is staged on its own.
        VecTile<RSW, LOAD == kLoadExact, TR> buf;
        const int64_t tf = t1 < n_full ? t1 : n_full;
        int64_t t = t0;
        if (t < tf) buf.load_full(a.in, t, lane);
        for (; t < tf; ++t) {
            wave_sync();                 // previous tile fully read
            buf.template store<LAYOUT>(a.in, tile, lane);
            wave_sync();                 // tile visible to every lane
            if (t + 1 < tf) buf.load_full(a.in, t + 1, lane);
            finish(t, body(t));
        }
        if (t < t1) {                         // t == n_full: the partial tile
            wave_sync();
            stage_now<XT, RS, LOAD, LAYOUT, TR>(a.in, tile, t, lane);
            wave_sync();
            finish(t, body(t));
        }
    } else {
        for (int64_t t = t0; t < t1; ++t) {
            wave_sync();
            stage_now<XT, RS, LOAD, LAYOUT, TR>(a.in, tile, t, lane);
            wave_sync();
            finish(t, body(t));
        }
    }
}

// LDS layout: [tables (if staged)] [one record tile per wavefront] [one result buffer per
// wavefront].  `tile` is the word view of this wavefront's tile (TR records).
template <int XT, int RS, int TR = kTileRows>
__device__ __forceinline__ void wave_buffers(const KArgs &a, char *after_tables, float *&tile,
                                             uint8_t *&obuf) {
    constexpr int kTileBytes = TR * row_words<XT, RS>() * 4;
    const int wave = threadIdx.x >> 6;
    tile = reinterpret_cast<float *>(after_tables + wave * kTileBytes);
    const int obytes = out_buffer_bytes(a.out_cap, a.out_kind == 0 ? 1 : 4, TR);
    obuf = reinterpret_cast<uint8_t *>(after_tables) + a.waves * kTileBytes + wave * obytes;
}

template <class T>
__device__ __forceinline__ void store_value(void *out, int out_kind, int64_t n, int64_t row,
                                            T v) {
    if (row < n) {
        if (out_kind == 0)
            static_cast<uint8_t *>(out)[row] = uint8_t(v);
        else
            static_cast<int32_t *>(out)[row] = int32_t(v);
    }
}

}  // namespace dev
}  // namespace dtree
