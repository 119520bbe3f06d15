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
// at most 128 VGPRs per lane as data (16 waves per CU); the
// float scans need more scratch registers and keep 64.  Small arrays want
// more, smaller tiles to occupy the 256 CUs.  Between 2^22 and 2^27 integer
// elements the 32768-element tile is faster than the 40960-element one
// (measured cold: 7.4 against 14.3 us at 2^22, 119 against 138 us at 2^26:
// the larger tile leaves CUs without a tile at the small end, and its fewer
// tiles fill the last round of workgroups unevenly).
struct GeomSmall { static constexpr int W = 4, J = 4; };   //  4096 elements
struct GeomMid { static constexpr int W = 4, J = 16; };    // 16384 elements
struct GeomBig { static constexpr int W = 8, J = 16; };    // 32768 elements
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

// --- the large-array kernel: register chunks plus LDS chunks per wave
//
// Same single pass, but each wave also owns L further 1 KB chunks that are
// loaded straight into LDS (global_load_lds_dwordx4, no VGPRs) and read back
// only for the chunk totals and for the stores.  Registers cap what a tile
// can hold while it waits for its predecessors; LDS adds 9 KB per wave, so
// the same number of tiles in flight carries 45 % more bytes.  Measured at
// n = 2^28: int32 420 -> 405 us, fp32 426 -> 410 us (two 8-wave workgroups
// per CU).  One 16-wave workgroup per CU (144 KB of LDS), with the same
// chunks per wave, halves the tiles and with them the tickets and the
// look-back chain: 402 -> 393 us (int32, 19 register chunks: 20 spill) and
// 410 -> 402 us (fp32); 4-wave workgroups, four per CU, took 428 us and
// 2-wave ones 479.  Wave w owns chunks [w*JT, (w+1)*JT) of the tile (JT = J+L),
// register chunks first.  Only full tiles take this path; a ragged last tile
// scans its elements in at most two passes of register-only sub-tiles, the
// first one loaded before its look-back (no tile waits on the last one).
template <class T, int J, int L, int WV>
struct LdsGeom {
    static constexpr int W = WV, JT = J + L;
    static constexpr int kThreads = W * kWave;
    static constexpr int64_t kElems = (int64_t)W * JT * kWave * 4;
};

template <class T, int J, int L, int WV, bool EXCL>
__global__ __launch_bounds__(WV * kWave) LS_OCCUPANCY4 void k_scan_lookback_lds(
    const T* x, T* y, int64_t n, WsHeader* hdr, uint64_t* status, int64_t status_words,
    uint32_t ntiles, const T* carry_in, T* total_out) {
    using G = LdsGeom<T, J, L, WV>;
    static_assert(G::kThreads == WV * kWave, "launch bounds");
    using Sub = Tile<T, T, 4, 16, G::W>;  // passes over a ragged last tile (65536 elements)
    static_assert(2 * Sub::kElems >= G::kElems, "a ragged tile takes at most two passes");
    __shared__ u32x4 s_buf[G::W * L * kWave];
    __shared__ Ticket s_ticket;
    __shared__ T s_wtot[G::W];
    __shared__ T s_carry;

    if (threadIdx.x == 0) s_ticket = take_ticket(hdr, ntiles);
    __syncthreads();
    const uint32_t tile32 = (uint32_t)__builtin_amdgcn_readfirstlane(s_ticket.tile);
    const uint32_t epoch = (uint32_t)__builtin_amdgcn_readfirstlane(s_ticket.epoch);
    if (tile32 >= ntiles) {  // only with a workspace that was never zero-filled
        if (threadIdx.x == 0)
            __hip_atomic_store(&hdr->error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return;
    }
    const int64_t base = (int64_t)tile32 * G::kElems;
    const T c0 = (tile32 == 0 && carry_in) ? *carry_in : T(0);
    const int w = threadIdx.x / kWave;
    const int lane = lane_id();

    if (base + G::kElems > n) {
        // Ragged last tile: register-only passes of Sub tiles (at most two).
        // The first pass is loaded before the look-back so that only its
        // stores wait for the predecessors; nothing waits on this tile, so
        // the aggregate it publishes (the first pass's) is never read.
        T v[Sub::J][4];
        Sub::template load<true>(x, n, base, v);
        const T wtot = Sub::template wave_scan<EXCL>(v);
        T wofs;
        const T agg0 = Sub::combine_waves(wtot, s_wtot, &wofs);
        if (threadIdx.x < kWave) {
            const T excl = lookback<T>(status, tile32, 0u, agg0, c0, epoch, hdr);
            if (threadIdx.x == 0) {
                s_carry = excl;
                finish_epoch(hdr, epoch, ntiles, status, status_words);
            }
        }
        __syncthreads();
        T carry = s_carry;
        Sub::template store<true>(y, n, base, v, carry + wofs);
        carry = carry + agg0;
        for (int64_t b = base + Sub::kElems; b < n; b += Sub::kElems) {
            Sub::template load<true>(x, n, b, v);
            const T wt = Sub::template wave_scan<EXCL>(v);
            T wo;
            const T agg = Sub::combine_waves(wt, s_wtot, &wo);
            Sub::template store<true>(y, n, b, v, carry + wo);
            carry = carry + agg;
            __syncthreads();  // s_wtot is rewritten by the next pass
        }
        if (total_out && threadIdx.x == 0) *total_out = carry;
        return;
    }

    const T* xw = x + base + (int64_t)w * (G::JT * kWave * 4);
    T* yw = y + base + (int64_t)w * (G::JT * kWave * 4);
    u32x4* lw = s_buf + w * L * kWave;
    T v[J][4];
    // Issue order: the LDS chunks, then the register chunks, then nothing
    // else until every load is in flight (the scheduling barriers keep the
    // compiler from interleaving scan work, which would make it wait for all
    // loads issued so far: it cannot count LDS-direct loads individually).
    // The register chunks load nontemporally (the input is read once); that
    // measured 404 against 411 us at n = 2^28, the same hint on the
    // LDS-direct loads 406.
#pragma unroll
    for (int c = 0; c < L; ++c)
        __builtin_amdgcn_global_load_lds((const void*)(xw + (J + c) * kWave * 4 + lane * 4),
                                         lw + c * kWave, 16, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = 0; j < J; ++j) load_vec<T, T, 4, true>(xw + j * kWave * 4 + lane * 4, v[j]);
    __builtin_amdgcn_sched_barrier(0);
    // register chunks: the tile scan of Tile::wave_scan
    const T run = Tile<T, T, 4, J, G::W>::template wave_scan<EXCL>(v);
    // LDS chunks: totals only (the data stays in LDS until the stores)
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    T lrun = T(0);
#pragma unroll
    for (int c = 0; c < L; ++c) {
        const u32x4 r = lw[c * kWave + lane];
        lrun = lrun + wave_sum(((Bits<T>::from(r.x) + Bits<T>::from(r.y)) +
                                Bits<T>::from(r.z)) + Bits<T>::from(r.w));
    }
    T wofs;
    const T agg = Tile<T, T, 4, J, G::W>::combine_waves(run + lrun, s_wtot, &wofs);
    if (threadIdx.x < kWave) {
        const T excl = lookback<T>(status, tile32, 0u, agg, c0, epoch, hdr);
        if (threadIdx.x == 0) {
            s_carry = excl;
            if (total_out && tile32 == ntiles - 1) *total_out = excl + agg;
            finish_epoch(hdr, epoch, ntiles, status, status_words);
        }
    }
    __syncthreads();
    const T carry = s_carry + wofs;
#pragma unroll
    for (int j = 0; j < J; ++j) {
        T o[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = carry + v[j][e];
        store_vec<T, 4>(yw + j * kWave * 4 + lane * 4, o);
    }
    T c2 = carry + run;
#pragma unroll
    for (int c = 0; c < L; ++c) {
        const u32x4 r = lw[c * kWave + lane];
        T p[4] = {Bits<T>::from(r.x), Bits<T>::from(r.y), Bits<T>::from(r.z), Bits<T>::from(r.w)};
#pragma unroll
        for (int e = 1; e < 4; ++e) p[e] = p[e - 1] + p[e];
        const T inc = wave_incl_scan(p[3]);
        const T lb = c2 + wave_shr1(inc);
        T o[4];
        if (EXCL) {
            o[0] = lb;
#pragma unroll
            for (int e = 1; e < 4; ++e) o[e] = lb + p[e - 1];
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) o[e] = lb + p[e];
        }
        store_vec<T, 4>(yw + (J + c) * kWave * 4 + lane * 4, o);
        c2 = c2 + lane_read(inc, kWave - 1);
    }
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
    TileT::template load<VEC, true>(x, n, base, v);
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
    TileT::template load<VEC, true>(x, n, base, v);
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

// Register + LDS tiles for the largest 32-bit arrays: 114688 (integer) or
// 102400 (float) elements per tile, one 16-wave workgroup per CU, the most
// that fits 128 VGPRs per lane without spilling and 160 KB of LDS.
template <class T>
struct LdsChunks {
    static constexpr int J = std::is_same<T, float>::value ? 16 : 19, L = 9, W = 16;
};

template <class T>
static void scan1d_lds(bool exclusive, const T* x, T* y, int64_t n, const T* carry_in,
                       T* total_out, WsHeader* hdr, uint64_t* status, int64_t status_words,
                       hipStream_t stream) {
    constexpr int J = LdsChunks<T>::J, L = LdsChunks<T>::L, WV = LdsChunks<T>::W;
    using G = LdsGeom<T, J, L, WV>;
    const uint32_t nt = (uint32_t)num_tiles(n, G::kElems);
    auto k = exclusive ? k_scan_lookback_lds<T, J, L, WV, true> : k_scan_lookback_lds<T, J, L, WV, false>;
    hipLaunchKernelGGL(k, dim3(nt), dim3(G::kThreads), 0, stream, x, y, n, hdr, status,
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
    else if (n >= (int64_t(1) << 27) && std::is_same<In, T>::value)
        scan1d_lds<T>(exclusive, reinterpret_cast<const T*>(x), y, n, carry_in, total_out, hdr,
                      status, status_words, stream);
    else if (n >= (int64_t(1) << 27))
        scan1d_geom<In, T, GeomLarge<T>, true>(exclusive, x, y, n, carry_in, total_out, hdr,
                                               status, status_words, stream);
    else if (n >= (int64_t(1) << 22))
        scan1d_geom<In, T, GeomBig, true>(exclusive, x, y, n, carry_in, total_out, hdr, status,
                                          status_words, stream);
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
    // fp16 inclusive scans of 2^27 elements and more run on the matrix cores:
    // measured against the wavefront tiles in one process (medians of 9
    // alternating rounds), 337.0 against 346.8 us at n = 2^28, 152.7 against
    // 153.7 us at 2^27, but slower below (79.0 against 80.1 us at 2^26, 28.9
    // against 29.6 at 2^24 cold, 10.2 against 11.0 at 2^22 cold).  The byte
    // scan on the matrix cores measured no faster (251 against 251 us at
    // 2^28), so byte scans stay on the wavefront tiles.
    if (kind == Kind::F16F32 && !exclusive && !carry_in && !total_out &&
        n >= (int64_t(1) << 27) && aligned(x, 16) && aligned(y, 4))
        return launch_scan1d_mfma_f16(reinterpret_cast<const uint16_t*>(x),
                                      reinterpret_cast<float*>(y), n, ws, ws_bytes, stream);
    return launch_scan1d_tiles(kind, exclusive, x, y, n, carry_in, total_out, ws, ws_bytes,
                               stream);
}

hipError_t launch_scan1d_tiles(Kind kind, bool exclusive, const void* x, void* y, int64_t n,
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

// Copy the header's error word to *out and, if `reset`, clear it.
__global__ void k_workspace_error(WsHeader* hdr, int32_t* out, int reset) {
    if (threadIdx.x == 0) {
        const uint32_t e = __hip_atomic_load(&hdr->error, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        *out = (int32_t)e;
        if (reset) __hip_atomic_store(&hdr->error, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

hipError_t launch_workspace_error(void* ws, int32_t* out, bool reset, hipStream_t stream) {
    hipLaunchKernelGGL(k_workspace_error, dim3(1), dim3(64), 0, stream,
                       reinterpret_cast<WsHeader*>(ws), out, reset ? 1 : 0);
    return hipGetLastError();
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
