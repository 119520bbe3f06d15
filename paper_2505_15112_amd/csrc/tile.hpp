// tile.hpp -- the workgroup tile shared by every scan kernel.
//
// A tile is WAVES wavefronts x J chunks x 64 lanes x V elements, laid out so
// that chunk j of wave w covers 64*V contiguous elements and lane l owns V
// contiguous elements of it:
//     element(w, j, l, e) = tile_base + ((w*J + j)*64 + l)*V + e.
// One chunk is therefore one fully coalesced vector load per lane (16 bytes
// for 32-bit data with V = 4), and a wave reads J*64*V contiguous elements.
// The tile scan is: serial scan of the V elements in each lane, a DPP
// wavefront scan of the 64 lane totals per chunk, a running carry over the J
// chunks of the wave, and the wave totals combined through LDS.
#pragma once

#include "device.hpp"

namespace ls {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// ---------------------------------------------------------------- conversion

template <class In, class T>
struct Conv;
template <>
struct Conv<uint32_t, uint32_t> {
    __device__ static uint32_t f(uint32_t v) { return v; }
};
template <>
struct Conv<int32_t, int32_t> {  // moved as-is (indices)
    __device__ static int32_t f(int32_t v) { return v; }
};
template <>
struct Conv<float, float> {
    __device__ static float f(float v) { return v; }
};
template <>
struct Conv<uint16_t, float> {  // IEEE binary16 bits -> fp32 (exact)
    __device__ static float f(uint16_t v) { return (float)__builtin_bit_cast(_Float16, v); }
};
template <>
struct Conv<uint8_t, uint32_t> {  // unsigned byte value
    __device__ static uint32_t f(uint8_t v) { return v; }
};

// Aligned vector load of V elements of In, converted to T.  NT: 16-byte
// loads are nontemporal (data read once, kept out of the caches' way).
template <class In, class T, int V, bool NT = false>
__device__ __forceinline__ void load_vec(const In* p, T (&out)[V]) {
    constexpr int kBytes = V * (int)sizeof(In);
    In e[V];
    if constexpr (kBytes == 16) {
        const u32x4 r = NT ? __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p))
                           : *reinterpret_cast<const u32x4*>(p);
        __builtin_memcpy(e, &r, 16);
    } else if constexpr (kBytes == 8) {
        const u32x2 r = *reinterpret_cast<const u32x2*>(p);
        __builtin_memcpy(e, &r, 8);
    } else if constexpr (kBytes == 4) {
        const uint32_t r = *reinterpret_cast<const uint32_t*>(p);
        __builtin_memcpy(e, &r, 4);
    } else {
        static_assert(kBytes == 16 || kBytes == 8 || kBytes == 4, "unsupported vector width");
    }
#pragma unroll
    for (int i = 0; i < V; ++i) out[i] = Conv<In, T>::f(e[i]);
}

// Aligned vector store of V 32-bit elements (V/4 16-byte stores).
template <class T, int V>
__device__ __forceinline__ void store_vec(T* p, const T (&v)[V]) {
    static_assert(sizeof(T) == 4 && V % 4 == 0, "16-byte stores of 32-bit elements");
#pragma unroll
    for (int q = 0; q < V / 4; ++q) {
        u32x4 r;
        __builtin_memcpy(&r, v + 4 * q, 16);
        __builtin_nontemporal_store(r, reinterpret_cast<u32x4*>(p) + q);
    }
}

// ---------------------------------------------------------------- the tile

template <class In_, class T_, int V_, int J_, int WAVES_>
struct Tile {
    using In = In_;
    using T = T_;
    static constexpr int V = V_;
    static constexpr int J = J_;
    static constexpr int WAVES = WAVES_;
    static constexpr int kThreads = WAVES * kWave;
    static constexpr int kElems = WAVES * J * kWave * V;

    // Offset of the lane's chunk-j elements from the tile base (< kElems, so
    // 32 bits: with the tile base pointer wave-uniform, loads and stores take
    // the scalar-base + 32-bit vector-offset form and no 64-bit addresses live
    // in vector registers).
    __device__ static uint32_t lane_offset(int j) {
        const uint32_t w = threadIdx.x / kWave;
        return ((w * J + (uint32_t)j) * kWave + (uint32_t)lane_id()) * V;
    }
    __device__ static int64_t offset(int64_t base, int j) { return base + lane_offset(j); }

    // Load the tile starting at `base`; elements at or past n read as zero.
    // NT: nontemporal 16-byte loads (see load_vec).
    template <bool VEC, bool NT = false>
    __device__ static void load(const In* x, int64_t n, int64_t base, T (&v)[J][V]) {
        const In* xt = x + base;  // wave-uniform
        if (VEC && base + kElems <= n) {  // uniform: all vector loads issued back to back
#pragma unroll
            for (int j = 0; j < J; ++j) load_vec<In, T, V, NT>(xt + lane_offset(j), v[j]);
        } else {
            // Ragged last tile (or unaligned data): per chunk, a lane with all
            // V elements in range loads them without per-element tests (one
            // vector load when aligned), a lane straddling the end loads
            // element by element.  Counts are 32-bit (valid <= kElems).
            const int32_t valid = (int32_t)(n - base < kElems ? n - base : kElems);
#pragma unroll
            for (int j = 0; j < J; ++j) {
                const int32_t off = (int32_t)lane_offset(j);
                const int32_t rem = valid - off;
                if (rem >= V) {  // one branch per chunk, not one predicate per element
                    if (VEC) {
                        load_vec<In, T, V, NT>(xt + off, v[j]);
                    } else {
#pragma unroll
                        for (int e = 0; e < V; ++e) v[j][e] = Conv<In, T>::f(xt[off + e]);
                    }
                } else {
#pragma unroll
                    for (int e = 0; e < V; ++e) v[j][e] = e < rem ? Conv<In, T>::f(xt[off + e]) : T(0);
                }
            }
        }
    }

    // Tile-local scan up to the wave: afterwards v[j][e] is the sum of the
    // wave's elements before (EXCL) or up to and including (inclusive) that
    // element, so the only thing left to add is one wave-uniform carry.
    // Lane-serial scan of the V elements, DPP wavefront scan of the lane
    // totals per chunk, running total over the J chunks.  Returns the wave's
    // total (uniform).
    template <bool EXCL>
    __device__ static T wave_scan(T (&v)[J][V]) {
        T run = T(0);
#pragma unroll
        for (int j = 0; j < J; ++j) {
#pragma unroll
            for (int e = 1; e < V; ++e) v[j][e] = v[j][e - 1] + v[j][e];
            const T inc = wave_incl_scan(v[j][V - 1]);
            const T lb = run + wave_shr1(inc);  // everything in the wave before this lane's chunk-j elements
            if (EXCL) {
#pragma unroll
                for (int e = V - 1; e > 0; --e) v[j][e] = lb + v[j][e - 1];
                v[j][0] = lb;
            } else {
#pragma unroll
                for (int e = 0; e < V; ++e) v[j][e] = lb + v[j][e];
            }
            run = run + lane_read(inc, kWave - 1);
        }
        return run;
    }

    // Sum of the lane's elements (no scan), for reductions.
    __device__ static T lane_sum(const T (&v)[J][V]) {
        T s = T(0);
#pragma unroll
        for (int j = 0; j < J; ++j)
#pragma unroll
            for (int e = 0; e < V; ++e) s = s + v[j][e];
        return s;
    }

    // Combine wave totals through LDS: returns the tile aggregate; *wofs gets
    // the sum of the waves before this one.  Contains a barrier.
    __device__ static T combine_waves(T wave_total, T* s_wtot, T* wofs) {
        const int w = threadIdx.x / kWave;
        if (lane_id() == 0) s_wtot[w] = wave_total;
        __syncthreads();
        if constexpr (WAVES > 8) {
            // Many waves: the wave totals are scanned across lanes instead of
            // summed by every lane in a loop, which holds one register per
            // wave total (and spills the 16-wave tiles).
            const T inc = wave_incl_scan(lane_id() < WAVES ? s_wtot[lane_id()] : T(0));
            const int wu = __builtin_amdgcn_readfirstlane(w);
            *wofs = wu > 0 ? lane_read(inc, wu - 1) : T(0);
            return lane_read(inc, WAVES - 1);
        }
        T before = T(0), agg = T(0);
#pragma unroll
        for (int k = 0; k < WAVES; ++k) {
            const T t = s_wtot[k];
            if (k < w) before = before + t;
            agg = agg + t;
        }
        *wofs = before;
        return agg;
    }

    // Store carry + v (v from wave_scan; carry uniform per wave); only i < n.
    template <bool VEC>
    __device__ static void store(T* y, int64_t n, int64_t base, const T (&v)[J][V], T carry) {
        T* yt = y + base;  // wave-uniform
        if (VEC && base + kElems <= n) {
#pragma unroll
            for (int j = 0; j < J; ++j) {
                T o[V];
#pragma unroll
                for (int e = 0; e < V; ++e) o[e] = carry + v[j][e];
                store_vec<T, V>(yt + lane_offset(j), o);
            }
        } else {
            const int32_t valid = (int32_t)(n - base < kElems ? n - base : kElems);
#pragma unroll
            for (int j = 0; j < J; ++j) {
                const int32_t off = (int32_t)lane_offset(j);
                const int32_t rem = valid - off;
                T o[V];
#pragma unroll
                for (int e = 0; e < V; ++e) o[e] = carry + v[j][e];
                if (rem >= V) {
                    if (VEC) {
                        store_vec<T, V>(yt + off, o);
                    } else {
#pragma unroll
                        for (int e = 0; e < V; ++e) yt[off + e] = o[e];
                    }
                } else {
#pragma unroll
                    for (int e = 0; e < V; ++e)
                        if (e < rem) yt[off + e] = o[e];
                }
            }
        }
    }
};

}  // namespace ls
