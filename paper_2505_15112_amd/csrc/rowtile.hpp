// rowtile.hpp -- what the row kernels share: the tile geometries for rows
// of a row-major rows x len matrix, and the per-row arrival counter with
// which a row's last tile to finish learns that it is the last.
#pragma once

#include "tile.hpp"

namespace ls {

constexpr int kRVec = 4;
constexpr int64_t kRowTile = 4096;  // rows up to this length: one wavefront per row

// Long-row tile geometries (waves x chunks x 64 x 4): long rows take big
// tiles (each tile costs one ticket, about 11 ns serialised on MI355X), rows
// of a few tiles take smaller ones so that a row still spans several tiles.
struct RGeomS { static constexpr int W = 4, J = 4; };   //  4096
struct RGeomM { static constexpr int W = 4, J = 8; };   //  8192
struct RGeomL { static constexpr int W = 8, J = 16; };  // 32768
inline int64_t row_tile(int64_t len) {
    return len > 65536 ? 32768 : (len > 16384 ? 8192 : 4096);
}
inline int64_t row_segments(int64_t len) { return (len + row_tile(len) - 1) / row_tile(len); }
// The same tile for misaligned rows (element-wise loads need more registers
// per element): twice the waves, half the chunks.
template <class T, class G, bool VEC>
using RowTile = Tile<T, T, kRVec, VEC ? G::J : G::J / 2, VEC ? G::W : G::W * 2>;
inline bool long_rows(int64_t len) { return len > kRowTile; }

// Row words in the workspace (a published tile sum, a row's arrival count)
// carry the top three bits 001.  Other ops leave status words with a
// non-zero state in the top two bits, or counts with the top three bits
// clear, and cleared words are 0, so nothing else can pass for such a word.
constexpr uint64_t kRowTag = 1ull << 61;
__device__ __forceinline__ bool row_word(uint64_t w) { return (w >> 61) == 1; }

// Count one arrival in the row's counter; returns the arrivals before it.  A
// word without the tag (left by another op sharing the workspace) counts as
// zero, hence compare-and-swap rather than a plain add.
__device__ __forceinline__ uint32_t row_arrive(uint64_t* counter) {
    adversarial_pause((uint32_t)(uintptr_t)counter);
    uint64_t old = __hip_atomic_load(counter, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    while (true) {
        const uint32_t before = row_word(old) ? (uint32_t)old : 0u;
        uint64_t expected = old;
        if (__hip_atomic_compare_exchange_strong(counter, &expected, kRowTag | (before + 1u),
                                                 __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                                 __HIP_MEMORY_SCOPE_AGENT))
            return before;
        old = expected;
    }
}

}  // namespace ls
