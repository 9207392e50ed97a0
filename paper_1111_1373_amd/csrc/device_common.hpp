// Device building blocks shared by the single-tree and forest kernels (gfx950).
//
// Record tiles: every wavefront owns a private tile of 64 records (one per lane) in the
// LDS.  Row r (record) starts at r*RS floats; column c is stored at position c ^ swz(r).
// The XOR spreads the 64 rows over all 64 banks for a fixed column, so the top levels of
// a tree (where every lane reads the same feature) are conflict-free, and the 16-byte
// staging stores land on distinct banks.
//
// Window tables (built on the host, see encode.hpp): for window w, slot h holds the
// (threshold, feature) of heap position h; exit e holds the next window (>= 0) or the
// result -(value + 1).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>

#include "kernels.hpp"

namespace dtree {
namespace dev {

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
// across this point.
__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ uint32_t div_f(uint32_t e, const Rows &in) {
    return in.n_features == 1 ? e : __umulhi(e, in.magic_f);
}

__device__ __forceinline__ int valid_rows(const Rows &in, int64_t tile) {
    const int64_t left = in.n - tile * kTileRows;
    return left < kTileRows ? int(left) : kTileRows;
}

// Store 4 consecutive features (c % 4 == 0) of row r into the swizzled tile.
template <int RS>
__device__ __forceinline__ void put4(float *tile, int r, int c, f32x4 v) {
    float *row = tile + r * RS;
    const int s = swz<RS>(r);
    row[(c + 0) ^ s] = v.x;
    row[(c + 1) ^ s] = v.y;
    row[(c + 2) ^ s] = v.z;
    row[(c + 3) ^ s] = v.w;
}

// Vectorised staging (ld == F, F % 4 == 0, 16-byte aligned base), one tile held in
// registers so that the next tile's loads overlap the walk of the current one.
template <int RS>
struct VecTile {
    static constexpr int kVec = RS / 4;   // 16-byte vectors per lane for F == RS
    f32x4 v[kVec];

    __device__ __forceinline__ void load(const Rows &in, int64_t tile, int lane) {
        const int nvec = (valid_rows(in, tile) * in.n_features) >> 2;
        const f32x4 *src = reinterpret_cast<const f32x4 *>(in.x + tile * kTileRows * in.n_features);
#pragma unroll
        for (int k = 0; k < kVec; ++k) {
            const int q = k * 64 + lane;
            v[k] = q < nvec ? __builtin_nontemporal_load(src + q) : f32x4{0.f, 0.f, 0.f, 0.f};
        }
    }

    __device__ __forceinline__ void store(const Rows &in, float *tile, int lane) const {
        const int full = kTileRows * in.n_features / 4;
#pragma unroll
        for (int k = 0; k < kVec; ++k) {
            const int q = k * 64 + lane;
            if (q < full) {
                const uint32_t e = uint32_t(q) * 4u;
                const int r = int(div_f(e, in));
                put4<RS>(tile, r, int(e) - r * in.n_features, v[k]);
            }
        }
    }
};

// Vectorised staging of wide rows (RS > 64) in chunks of 16 vectors per lane.
template <int RS>
__device__ __forceinline__ void stage_wide(const Rows &in, float *tile, int64_t t, int lane) {
    const int nvec = (valid_rows(in, t) * in.n_features) >> 2;
    const int full = kTileRows * in.n_features / 4;
    const f32x4 *src = reinterpret_cast<const f32x4 *>(in.x + t * kTileRows * in.n_features);
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
                const int r = int(div_f(e, in));
                put4<RS>(tile, r, int(e) - r * in.n_features, v[k]);
            }
        }
    }
}

// General staging: any ld >= F, any 4-byte alignment.
template <int RS>
__device__ __forceinline__ void stage_scalar(const Rows &in, float *tile, int64_t t, int lane) {
    const int64_t row0 = t * kTileRows;
    const int valid = valid_rows(in, t);
    for (int k = 0; k < in.n_features; ++k) {
        const uint32_t idx = uint32_t(k * 64 + lane);
        const int r = int(div_f(idx, in));
        const int c = int(idx) - r * in.n_features;
        float v = 0.f;
        if (r < valid) v = in.x[(row0 + r) * in.ld + c];
        tile[r * RS + (c ^ swz<RS>(r))] = v;
    }
}

// Stage tile t without register prefetch.
template <int RS, bool VEC>
__device__ __forceinline__ void stage_now(const Rows &in, float *tile, int64_t t, int lane) {
    if constexpr (VEC && RS <= 64) {
        VecTile<RS> buf;
        buf.load(in, t, lane);
        buf.store(in, tile, lane);
    } else if constexpr (VEC) {
        stage_wide<RS>(in, tile, t, lane);
    } else {
        stage_scalar<RS>(in, tile, t, lane);
    }
}

// ---- data decomposition: the record of this lane walks one tree --------------------------
// Within a window: h <- 2h + 1 + !(x[f_h] < t_h) for exactly D steps (Procedure 2's
// child + predicate step in heap form); then the exit names the next window or the result.
__device__ __forceinline__ int32_t walk_data(const Slot *slots, const int32_t *exits, int D,
                                             int levels, const float *row, int sw) {
    const int last = (1 << D) - 1;
    int w = 0;
    int32_t code = -1;
    for (int level = 0; level < levels; ++level) {
        const int base = w << D;
        int h = 0;
        for (int k = 0; k < D; ++k) {
            const Slot s = slots[base + h];
            const float xv = row[s.f ^ sw];
            h = 2 * h + 1 + int(!(xv < s.t));
        }
        code = exits[base + h - last];
        if (code < 0) break;
        w = code;
    }
    return code;
}

// ---- speculative decomposition: a tile of 64 records through one tree -------------------
// A segment of S = 2^D lanes is the record group of one record: lane j evaluates heap slot
// j of the record's current window (the processor-node map of Procedure 5), so one
// wavefront instruction evaluates 64/S records' windows.  One ballot gathers the 64
// outcomes; record r's segment is handed to lane r, which walks its bits from the window
// root to the exit.
template <int RS, int D>
struct Spec {
    static constexpr int S = 1 << D;
    using Bits = typename std::conditional<(S > 32), uint64_t, uint32_t>::type;
    int j;          // slot evaluated by this lane
    int seg_shift;  // first lane of this lane's segment

    __device__ __forceinline__ explicit Spec(int lane)
        : j(lane & (S - 1)), seg_shift(lane & ~(S - 1)) {}

    // One window level for the 64 records.  In round g, the segment starting at lane b
    // evaluates record b + g, so record r's bits arrive in r's own segment in the round
    // g == r % S.
    __device__ __forceinline__ Bits eval(const Slot *slots, bool first, const Slot &root, int w,
                                         const float *tile) const {
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
    }

    __device__ __forceinline__ int walk(Bits bits) const {
        int h = 0;
#pragma unroll
        for (int k = 0; k < D; ++k) h = 2 * h + 1 + int((bits >> h) & 1);
        return h - (S - 1);
    }

    // Exit code of every lane's record.  `root` = slots[j] of window 0.  All 64 lanes
    // must be active.
    __device__ __forceinline__ int32_t run(const Slot *slots, const int32_t *exits, int levels,
                                           const Slot &root, const float *tile) const {
        int w = 0;
        int32_t code = exits[walk(eval(slots, true, root, 0, tile))];
        bool done = code < 0;
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
};

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
