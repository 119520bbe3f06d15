// scan1d.hip -- 1-D prefix sums (Section 2 definition; exclusive form of the
// appendix "Exclusive and int8 scan").
//
// Primary path: one kernel, single pass over HBM (n reads + n writes, the
// 2N-transfer bound of Section 2.1), carries propagated between tiles by
// decoupled look-back on packed, epoch-tagged status words in the caller's
// workspace (which therefore needs no clearing between calls).
//
// Check path (reduce-then-scan, Section 2.1's RSS strategy and the two phases
// of Algorithm 3): per-tile sums, one workgroup scanning the tile sums, then
// every tile rescanned with its carry -- 3N transfers, no inter-workgroup
// waiting at all.
#include <type_traits>

#include "launch.hpp"
#include "tile.hpp"

namespace ls {

// Tile geometries (waves x chunks x 64 lanes x 4 elements).  Every tile costs
// one ticket and one look-back, so big arrays want big tiles: measured on
// MI355X at n = 2^28, 4096-element tiles reach half the device memcpy rate
// and 32768-element tiles match it.  A tile's data stays in registers from
// its loads until its stores, so the bytes in flight per CU are set by how
// much of the register file holds data: the large integer tile keeps 80 of
// at most 128 VGPRs per lane as data (two 8-wave workgroups per CU); the
// float scans need more scratch registers and keep 64.  Small arrays want
// more, smaller tiles to occupy the 256 CUs.
struct GeomSmall { static constexpr int W = 4, J = 4; };   //  4096 elements
struct GeomMid { static constexpr int W = 4, J = 16; };    // 16384 elements
template <class T>
struct GeomLarge {  // 40960 (integer) / 32768 (float) elements
    static constexpr int W = 8, J = std::is_same<T, float>::value ? 16 : 20;
};
// Misaligned data is loaded element by element: more registers per element,
// so fewer elements per lane.
struct GeomUnaligned { static constexpr int W = 8, J = 8; };  // 16384 elements
constexpr int kVec = 4;
constexpr int64_t kMinTileElems = GeomSmall::W * GeomSmall::J * kWave * kVec;
constexpr int64_t kRssTileElems = GeomMid::W * GeomMid::J * kWave * kVec;

// Workspaces are sized for the smallest tile, so any geometry fits.
static inline int64_t num_tiles(int64_t n, int64_t tile) { return (n + tile - 1) / tile; }

// ---------------------------------------------------------------- kernels

template <class T>
__global__ void k_write_total(T* total_out, const T* carry_in) {
    if (threadIdx.x == 0) *total_out = carry_in ? *carry_in : T(0);
}

template <class TileT, bool EXCL, bool VEC>
__global__ __launch_bounds__(TileT::kThreads) LS_OCCUPANCY4 void k_scan_lookback(
    const typename TileT::In* x, typename TileT::T* y, int64_t n, WsHeader* hdr,
    uint64_t* status, int64_t status_words, uint32_t ntiles, const typename TileT::T* carry_in,
    typename TileT::T* total_out) {
    using T = typename TileT::T;
    __shared__ Ticket s_ticket;
    __shared__ T s_wtot[TileT::WAVES];
    __shared__ T s_carry;

    if (threadIdx.x == 0) s_ticket = take_ticket(hdr, ntiles);
    __syncthreads();
    // wave-uniform from here on
    const uint32_t tile32 = (uint32_t)__builtin_amdgcn_readfirstlane(s_ticket.tile);
    const uint32_t epoch = (uint32_t)__builtin_amdgcn_readfirstlane(s_ticket.epoch);
    if (tile32 >= ntiles) {  // only with a workspace that was never zero-filled
        if (threadIdx.x == 0)
            __hip_atomic_store(&hdr->error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return;
    }
    const int64_t tile = tile32;
    const int64_t base = tile * TileT::kElems;

    T v[TileT::J][TileT::V];
    TileT::template load<VEC>(x, n, base, v);
    const T wtot = TileT::template wave_scan<EXCL>(v);
    T wofs;
    const T agg = TileT::combine_waves(wtot, s_wtot, &wofs);

    if (threadIdx.x < kWave) {
        const T c0 = (tile == 0 && carry_in) ? *carry_in : T(0);
        const T excl = lookback<T>(status, tile32, 0u, agg, c0, epoch, hdr);
        if (threadIdx.x == 0) {
            s_carry = excl;
            if (total_out && tile == ntiles - 1) *total_out = excl + agg;
            finish_epoch(hdr, epoch, ntiles, status, status_words);
        }
    }
    __syncthreads();
    TileT::template store<VEC>(y, n, base, v, s_carry + wofs);
}

// --- reduce-then-scan

template <class TileT, bool VEC>
__global__ __launch_bounds__(TileT::kThreads) LS_OCCUPANCY4 void k_rss_reduce(const typename TileT::In* x,
                                                                int64_t n,
                                                                typename TileT::T* partial) {
    using T = typename TileT::T;
    __shared__ T s_wtot[TileT::WAVES];
    const int64_t base = (int64_t)blockIdx.x * TileT::kElems;
    T v[TileT::J][TileT::V];
    TileT::template load<VEC>(x, n, base, v);
    const T wtot = wave_sum(TileT::lane_sum(v));
    T wofs;
    const T agg = TileT::combine_waves(wtot, s_wtot, &wofs);
    if (threadIdx.x == 0) partial[blockIdx.x] = agg;
}

// One workgroup of 1024 threads: exclusive scan of the tile sums in place.
template <class T>
__global__ __launch_bounds__(1024) void k_rss_spine(T* partial, int64_t ntiles) {
    constexpr int kW = 1024 / kWave;
    constexpr int kPer = 4;
    __shared__ T s_wtot[kW];
    const int lane = lane_id();
    const int w = threadIdx.x / kWave;
    T carry = T(0);
    for (int64_t b = 0; b < ntiles; b += 1024 * kPer) {
        T v[kPer];
        const int64_t off = b + (int64_t)threadIdx.x * kPer;
#pragma unroll
        for (int e = 0; e < kPer; ++e) v[e] = off + e < ntiles ? partial[off + e] : T(0);
        T s = T(0);
#pragma unroll
        for (int e = 0; e < kPer; ++e) s = s + v[e];
        const T inc = wave_incl_scan(s);
        const T lane_excl = wave_shr1(inc);
        if (lane == 0) s_wtot[w] = lane_read(inc, kWave - 1);
        __syncthreads();
        T wofs = T(0), tot = T(0);
        for (int k = 0; k < kW; ++k) {
            const T t = s_wtot[k];
            if (k < w) wofs = wofs + t;
            tot = tot + t;
        }
        T run = carry + wofs + lane_excl;
#pragma unroll
        for (int e = 0; e < kPer; ++e) {
            if (off + e < ntiles) partial[off + e] = run;
            run = run + v[e];
        }
        carry = carry + tot;
        __syncthreads();
    }
}

template <class TileT, bool VEC>
__global__ __launch_bounds__(TileT::kThreads) LS_OCCUPANCY4 void k_rss_rescan(const typename TileT::In* x,
                                                                typename TileT::T* y, int64_t n,
                                                                typename TileT::T* partial) {
    using T = typename TileT::T;
    __shared__ T s_wtot[TileT::WAVES];
    const int64_t base = (int64_t)blockIdx.x * TileT::kElems;
    const T carry = partial[blockIdx.x];
    T v[TileT::J][TileT::V];
    TileT::template load<VEC>(x, n, base, v);
    const T wtot = TileT::template wave_scan<false>(v);
    T wofs;
    TileT::combine_waves(wtot, s_wtot, &wofs);  // barrier: every thread has read `carry`
    // Leave the workspace zero where no status word is live, so that any
    // later look-back call can use it without clearing.
    if (threadIdx.x == 0) partial[blockIdx.x] = T(0);
    TileT::template store<VEC>(y, n, base, v, carry + wofs);
}

// ---------------------------------------------------------------- launchers

size_t scan1d_ws_bytes(int64_t n) {
    return kWsHeader + (size_t)num_tiles(n, kMinTileElems) * sizeof(uint64_t);
}

size_t scan1d_rss_ws_bytes(int64_t n) {
    return kWsHeader + (size_t)num_tiles(n, kRssTileElems) * sizeof(uint32_t);
}

static bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

template <class In, class T, class G, bool VEC>
static void scan1d_geom(bool exclusive, const In* x, T* y, int64_t n, const T* carry_in,
                        T* total_out, WsHeader* hdr, uint64_t* status, int64_t status_words,
                        hipStream_t stream) {
    using TileT = Tile<In, T, kVec, G::J, G::W>;
    const uint32_t nt = (uint32_t)num_tiles(n, TileT::kElems);
    auto k = exclusive ? k_scan_lookback<TileT, true, VEC> : k_scan_lookback<TileT, false, VEC>;
    hipLaunchKernelGGL(k, dim3(nt), dim3(TileT::kThreads), 0, stream, x, y, n, hdr, status,
                       status_words, nt, carry_in, total_out);
}

template <class In, class T>
static hipError_t scan1d_typed(bool exclusive, const In* x, T* y, int64_t n, const T* carry_in,
                               T* total_out, void* ws, size_t ws_bytes, hipStream_t stream) {
    if (n == 0) {
        if (total_out) hipLaunchKernelGGL(k_write_total<T>, dim3(1), dim3(64), 0, stream, total_out, carry_in);
        return hipGetLastError();
    }
    WsHeader* hdr = reinterpret_cast<WsHeader*>(ws);
    uint64_t* status = reinterpret_cast<uint64_t*>(reinterpret_cast<char*>(ws) + kWsHeader);
    const int64_t status_words = (int64_t)((ws_bytes - kWsHeader) / sizeof(uint64_t));
    // 16-byte vector loads and stores need both arrays 16-byte aligned.
    const bool vec = aligned(x, kVec * sizeof(In)) && aligned(y, kVec * sizeof(T));
    if (!vec && n >= (int64_t(1) << 18))
        scan1d_geom<In, T, GeomUnaligned, false>(exclusive, x, y, n, carry_in, total_out, hdr,
                                                 status, status_words, stream);
    else if (!vec)
        scan1d_geom<In, T, GeomSmall, false>(exclusive, x, y, n, carry_in, total_out, hdr, status,
                                             status_words, stream);
    else if (n >= (int64_t(1) << 22))
        scan1d_geom<In, T, GeomLarge<T>, true>(exclusive, x, y, n, carry_in, total_out, hdr,
                                               status, status_words, stream);
    else if (n >= (int64_t(1) << 18))
        scan1d_geom<In, T, GeomMid, true>(exclusive, x, y, n, carry_in, total_out, hdr, status,
                                          status_words, stream);
    else
        scan1d_geom<In, T, GeomSmall, true>(exclusive, x, y, n, carry_in, total_out, hdr, status,
                                            status_words, stream);
    return hipGetLastError();
}

hipError_t launch_scan1d(Kind kind, bool exclusive, const void* x, void* y, int64_t n,
                         const void* carry_in, void* total_out, void* ws, size_t ws_bytes,
                         hipStream_t stream) {
    switch (kind) {
        case Kind::I32:
            return scan1d_typed<uint32_t, uint32_t>(exclusive, (const uint32_t*)x, (uint32_t*)y, n,
                                                    (const uint32_t*)carry_in,
                                                    (uint32_t*)total_out, ws, ws_bytes, stream);
        case Kind::F32:
            return scan1d_typed<float, float>(exclusive, (const float*)x, (float*)y, n,
                                              (const float*)carry_in, (float*)total_out, ws,
                                              ws_bytes, stream);
        case Kind::F16F32:
            return scan1d_typed<uint16_t, float>(exclusive, (const uint16_t*)x, (float*)y, n,
                                                 (const float*)carry_in, (float*)total_out, ws,
                                                 ws_bytes, stream);
        case Kind::U8I32:
            return scan1d_typed<uint8_t, uint32_t>(exclusive, (const uint8_t*)x, (uint32_t*)y, n,
                                                   (const uint32_t*)carry_in,
                                                   (uint32_t*)total_out, ws, ws_bytes, stream);
    }
    return hipErrorInvalidValue;
}

template <class In, class T>
static hipError_t rss_typed(const In* x, T* y, int64_t n, void* ws, hipStream_t stream) {
    using TV = Tile<In, T, kVec, GeomMid::J, GeomMid::W>;
    using TU = Tile<In, T, kVec, GeomUnaligned::J, GeomUnaligned::W>;  // misaligned data
    static_assert(TV::kElems == kRssTileElems && TU::kElems == kRssTileElems, "rss tile");
    if (n == 0) return hipSuccess;
    const int64_t nt = num_tiles(n, kRssTileElems);
    T* partial = reinterpret_cast<T*>(reinterpret_cast<char*>(ws) + kWsHeader);
    const bool vec = aligned(x, kVec * sizeof(In)) && aligned(y, kVec * sizeof(T));
    const dim3 grid((unsigned)nt), bv(TV::kThreads), bu(TU::kThreads);
    if (vec)
        hipLaunchKernelGGL((k_rss_reduce<TV, true>), grid, bv, 0, stream, x, n, partial);
    else
        hipLaunchKernelGGL((k_rss_reduce<TU, false>), grid, bu, 0, stream, x, n, partial);
    hipLaunchKernelGGL(k_rss_spine<T>, dim3(1), dim3(1024), 0, stream, partial, nt);
    if (vec)
        hipLaunchKernelGGL((k_rss_rescan<TV, true>), grid, bv, 0, stream, x, y, n, partial);
    else
        hipLaunchKernelGGL((k_rss_rescan<TU, false>), grid, bu, 0, stream, x, y, n, partial);
    return hipGetLastError();
}

hipError_t launch_scan1d_rss(Kind kind, const void* x, void* y, int64_t n, void* ws,
                             hipStream_t stream) {
    switch (kind) {
        case Kind::I32:
            return rss_typed<uint32_t, uint32_t>((const uint32_t*)x, (uint32_t*)y, n, ws, stream);
        case Kind::F32:
            return rss_typed<float, float>((const float*)x, (float*)y, n, ws, stream);
        default:
            return hipErrorInvalidValue;
    }
}

}  // namespace ls

namespace ls {

__global__ void k_fill_zero(uint64_t* p, int64_t words) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < words; i += stride) p[i] = 0;
}

hipError_t launch_workspace_init(void* ws, size_t ws_bytes, hipStream_t stream) {
    const int64_t words = (int64_t)(ws_bytes / sizeof(uint64_t));
    if (words == 0) return hipSuccess;
    const int64_t blocks = (words + 255) / 256;
    hipLaunchKernelGGL(k_fill_zero, dim3((unsigned)(blocks < 2048 ? blocks : 2048)), dim3(256), 0,
                       stream, reinterpret_cast<uint64_t*>(ws), words);
    return hipGetLastError();
}

}  // namespace ls
