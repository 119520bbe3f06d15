// rows.hip -- batched scans over the rows of a row-major rows x len matrix
// (appendix "Multiple (Batched) Scans") and the top-p cutoff built on them
// (Section 5 "Top-p or Nucleus Sampling").
//
// Two schedules, after the paper's observation that many short rows and a
// few long rows want different mappings (its batched-scan crossover):
//  * len <= one tile: one wavefront owns a whole row and walks it in chunks
//    of 64 lanes x 4 elements with a running carry -- many rows per
//    workgroup, no inter-workgroup communication;
//  * longer rows: each row is cut into tile-sized segments, tiles are handed
//    out row-major by ticket, and the decoupled look-back runs inside a row
//    (it stops at the row's first segment), so 128 rows of 2^17 still give
//    4096 workgroups to fill 256 CUs.
// The top-p cutoff needs only one index per row: every tile sums its part of
// the row and the row's last tile to finish locates the index (k_topp).
// Weighted sampling of rows up to 2^22 and the cutoff of rows up to 2^20 run
// as two kernels instead (tile sums, then one workgroup per row), with no
// per-row arrival.
#include <limits.h>

#include "launch.hpp"
#include "rowtile.hpp"

namespace ls {

// Wavefront minimum with DPP (lanes outside the row / disabled read INT_MAX).
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ int32_t dpp_min(int32_t v) {
    const int32_t o = __builtin_amdgcn_update_dpp(INT_MAX, v, CTRL, ROW_MASK, 0xf, false);
    return o < v ? o : v;
}
__device__ __forceinline__ int32_t wave_min(int32_t v) {
    v = dpp_min<0x111, 0xf>(v);
    v = dpp_min<0x112, 0xf>(v);
    v = dpp_min<0x114, 0xf>(v);
    v = dpp_min<0x118, 0xf>(v);
    v = dpp_min<0x142, 0xa>(v);
    v = dpp_min<0x143, 0xc>(v);
    return __builtin_amdgcn_readlane(v, kWave - 1);
}

// ---------------------------------------------------------------- rows of one tile

// Rows of 1025 to 4096 elements (a scan, not the top-p cutoff): one
// workgroup per row, the whole row one tile (4 waves of 4 chunks of 64 lanes
// x 4 when aligned), scanned in registers and stored; nothing crosses
// workgroups.  A wavefront per row walks such a row in up to 16 dependent
// steps; four waves take 4 each.  (The 128 x 4096 count tables of the row
// sort: 7.7 against ~4 us per scan.)
constexpr int64_t kRowsTileMin = 1024;
template <class TileT, bool EXCL, bool VEC>
__global__ __launch_bounds__(TileT::kThreads) LS_OCCUPANCY4 void k_rows_tile(
    const typename TileT::T* x, typename TileT::T* y, int64_t len) {
    using T = typename TileT::T;
    __shared__ T s_wtot[TileT::WAVES];
    const int64_t row = blockIdx.x;
    T v[TileT::J][TileT::V];
    TileT::template load<VEC>(x + row * len, len, 0, v);
    const T wtot = TileT::template wave_scan<EXCL>(v);
    T wofs;
    TileT::combine_waves(wtot, s_wtot, &wofs);
    TileT::template store<VEC>(y + row * len, len, 0, v, wofs);
}

// ---------------------------------------------------------------- long rows

template <class TileT, bool EXCL, bool VEC>
__global__ __launch_bounds__(TileT::kThreads) LS_OCCUPANCY4 void k_rows_lookback(
    const typename TileT::T* x, typename TileT::T* y, int64_t len, uint32_t segs,
    uint32_t ntiles, WsHeader* hdr, uint64_t* status, int64_t status_words) {
    using T = typename TileT::T;
    __shared__ Ticket s_ticket;
    __shared__ T s_wtot[TileT::WAVES];
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
    const uint32_t row32 = tile32 / segs;  // 32-bit: no 64-bit division code
    const int64_t row = row32;
    const int64_t seg = tile32 - row32 * segs;
    const int64_t base = seg * TileT::kElems;

    T v[TileT::J][TileT::V];
    TileT::template load<VEC, true>(x + row * len, len, base, v);  // read once: nontemporal
    const T wtot = TileT::template wave_scan<EXCL>(v);
    T wofs;
    const T agg = TileT::combine_waves(wtot, s_wtot, &wofs);

    if (threadIdx.x < kWave) {
        const T excl = lookback<T>(status, tile32, row32 * segs, agg, T(0), epoch, hdr);
        if (threadIdx.x == 0) {
            s_carry = excl;
            finish_epoch(hdr, epoch, ntiles, status, status_words);
        }
    }
    __syncthreads();
    TileT::template store<VEC>(y + row * len, len, base, v, s_carry + wofs);
}

// ---------------------------------------------------------------- top-p

// One kernel; no workgroup waits for another's work.  Every tile of a row
// sums its values, stores the sum (in a workspace word with its two top bits
// clear, which any look-back reads as "nothing published", and a "set" bit
// below them) and counts itself in the row's arrival counter.  The row's last
// tile to arrive -- every other tile has stored its sum by then, it waits only
// for the stores to become visible -- finishes the row from the tile sums and
// at most two re-read tiles (just read, so still in the 256 MB Infinity
// Cache), then clears the sums and the counter, so the workspace needs no
// clearing.  Three modes:
//  * cutoff (Section 5 "Top-p"): the first index whose running sum reaches p,
//    len - 1 if none -- the first tile whose inclusive sum reaches p, then
//    the index inside it (the two phases of the paper's Algorithm 3, MCScan,
//    with the down-sweep cut to the one tile that matters);
//  * weighted sample (appendix "Weighted Sampling"): the first index whose
//    running sum exceeds theta * W, W the row total;
//  * top-p sample: the cutoff k, then the first index j <= k whose running
//    sum exceeds theta * C_k, reported through `idx` (the source index of
//    each sorted position; null: j itself).
enum class ToppMode { Cutoff, Weighted, Sample };

__device__ __forceinline__ float topp_sum(const uint64_t* w) {
    return Bits<float>::from((uint32_t)__hip_atomic_load(w, __ATOMIC_RELAXED,
                                                         __HIP_MEMORY_SCOPE_AGENT));
}

// Wave 0 of the last workgroup: the sum of the row's tile sums, in order.
__device__ __forceinline__ float topp_total(const uint64_t* rs, uint32_t segs) {
    float carry = 0.f;
    for (uint32_t b = 0; b < segs; b += kWave) {
        const uint32_t s = b + lane_id();
        carry = carry + wave_sum(s < segs ? topp_sum(&rs[s]) : 0.f);
    }
    return carry;
}

// Wave 0 of the last workgroup: the first tile t < limit whose inclusive sum
// reaches `thr` (strict: exceeds it), in tile order; -1 if none.  *excl gets
// the sum of the tiles before t (or of all `limit` tiles when none).
__device__ __forceinline__ int32_t topp_find_tile(const uint64_t* rs, uint32_t limit, float thr,
                                                  bool strict, float* excl) {
    const int lane = lane_id();
    float carry = 0.f;
    for (uint32_t b = 0; b < limit; b += kWave) {
        const uint32_t s = b + lane;
        const float a = s < limit ? topp_sum(&rs[s]) : 0.f;
        const float inc = carry + wave_incl_scan(a);
        const uint64_t hit = __ballot(s < limit && (strict ? inc > thr : inc >= thr));
        if (hit) {
            const int l = __builtin_ctzll(hit);
            *excl = l ? lane_read(inc, l - 1) : carry;
            return (int32_t)(b + l);
        }
        carry = lane_read(inc, kWave - 1);
    }
    *excl = carry;
    return -1;
}

// The whole workgroup: load the tile at `base`, and find its first index
// i <= lim whose running sum (excl + the tile prefix) reaches `thr` (STRICT:
// exceeds it); none (rounding): the tile's last index, capped at lim.
// Returns the index; `val` gets the running sum there.  Offsets inside the
// tile are 32-bit, and each lane keeps only the running sums at its candidate
// and at the cap, so the tile's registers die with the search loop.
template <class TileT, bool VEC, bool STRICT, bool NEED_VAL>
__device__ __forceinline__ int64_t topp_find_in_tile(const float* xr, int64_t len, int64_t base,
                                                     float excl, float thr, int64_t lim,
                                                     float* s_wtot, int32_t* s_min, float* s_val,
                                                     float& val, bool& hit) {
    float v[TileT::J][TileT::V];
    float wofs;
    TileT::template load<VEC>(xr, len, base, v);
    TileT::combine_waves(TileT::template wave_scan<false>(v), s_wtot, &wofs);
    const float c = excl + wofs;
    const int64_t last = (base + TileT::kElems < len ? base + TileT::kElems : len) - 1;
    const int32_t cap = (int32_t)((last < lim ? last : lim) - base);  // in-tile, >= 0
    int32_t cand = INT_MAX;
    float cand_val = 0.f, cap_val = 0.f;
    bool has_cap = false;
#pragma unroll
    for (int j = TileT::J - 1; j >= 0; --j) {
        const int32_t off = (int32_t)TileT::lane_offset(j);
#pragma unroll
        for (int e = TileT::V - 1; e >= 0; --e) {
            const float run = c + v[j][e];
            if (off + e <= cap && (STRICT ? run > thr : run >= thr)) {
                cand = off + e;
                if (NEED_VAL) cand_val = run;
            }
            if (NEED_VAL && off + e == cap) {
                cap_val = run;
                has_cap = true;
            }
        }
    }
    const int32_t wm = wave_min(cand);
    if (lane_id() == 0) s_min[threadIdx.x / kWave] = wm;
    __syncthreads();
    int32_t m = INT_MAX;
    for (int k = 0; k < TileT::WAVES; ++k) m = s_min[k] < m ? s_min[k] : m;
    const int32_t f = m != INT_MAX ? m : cap;
    hit = m != INT_MAX;
    // exactly one lane holds the winner (or, with none, the cap)
    if (NEED_VAL) {
        if (m != INT_MAX ? cand == m : has_cap) *s_val = m != INT_MAX ? cand_val : cap_val;
        __syncthreads();
        val = *s_val;
    }
    __syncthreads();  // s_min / s_val free for the next call
    return base + f;
}

// topp_find_in_tile over the tile at `base`; when the running sum is needed
// and the tile is large, over its two halves in turn (the second only when
// the first holds no hit and the range goes on), so that half a tile of
// registers is live at a time.
template <class TileT, bool VEC, bool STRICT, bool NEED_VAL>
__device__ __forceinline__ int64_t topp_find(const float* xr, int64_t len, int64_t base,
                                             float excl, float thr, int64_t lim, float* s_wtot,
                                             int32_t* s_min, float* s_val, float& val) {
    bool hit;
    if constexpr (NEED_VAL && TileT::J > 8) {
        using H = Tile<float, float, TileT::V, TileT::J / 2, TileT::WAVES>;
        const int64_t f = topp_find_in_tile<H, VEC, STRICT, true>(xr, len, base, excl, thr, lim,
                                                                  s_wtot, s_min, s_val, val, hit);
        if (hit || f != base + H::kElems - 1 || f >= lim || f + 1 >= len) return f;
        return topp_find_in_tile<H, VEC, STRICT, true>(xr, len, base + H::kElems, val, thr, lim,
                                                       s_wtot, s_min, s_val, val, hit);
    } else {
        return topp_find_in_tile<TileT, VEC, STRICT, NEED_VAL>(xr, len, base, excl, thr, lim,
                                                               s_wtot, s_min, s_val, val, hit);
    }
}

template <class TileT, bool VEC, ToppMode MODE>
__global__ __launch_bounds__(TileT::kThreads) LS_OCCUPANCY4 void k_topp(
    const float* probs, const int32_t* idx, const float* theta, int32_t* cutoff, int32_t* token,
    int64_t len, uint32_t segs, float p, WsHeader* hdr, uint64_t* sums, uint64_t* arrivals) {
    __shared__ float s_wtot[TileT::WAVES];
    __shared__ uint32_t s_last;
    __shared__ int32_t s_tile;
    __shared__ float s_excl;
    __shared__ float s_thr;
    __shared__ int32_t s_min[TileT::WAVES];
    __shared__ float s_val;

    const uint32_t row32 = blockIdx.x / segs;
    const uint32_t seg = blockIdx.x - row32 * segs;
    const int64_t row = row32;
    const float* xr = probs + row * len;
    {
        float v[TileT::J][TileT::V];
        // weighted sampling reads the rows once (nontemporal); the top-p modes
        // re-read a tile or two at the end, which measured faster cached
        TileT::template load<VEC, MODE == ToppMode::Weighted>(xr, len, (int64_t)seg * TileT::kElems, v);
        float wofs;
        const float agg = TileT::combine_waves(wave_sum(TileT::lane_sum(v)), s_wtot, &wofs);
        if (threadIdx.x == 0) {
            // Relaxed only (a release/acquire pair at device scope would write
            // back and invalidate L2 in every workgroup): the sum word carries
            // its own "published" bit, and the last arrival waits for it.
            __hip_atomic_store(&sums[blockIdx.x], kRowTag | Bits<float>::to(agg),
                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            // Arrive only once the store is acknowledged: an agent-scope
            // store is written through to the level every CU reads at agent
            // scope, so the last arrival can never find an older word (one a
            // different op left in the workspace) in place of this sum.
            __builtin_amdgcn_s_waitcnt(0);
            s_last = row_arrive(&arrivals[row]) == segs - 1;
        }
    }
    __syncthreads();
    if (!s_last) return;  // uniform over the workgroup

    uint64_t* rs = sums + (int64_t)row32 * segs;
    const float th = MODE == ToppMode::Cutoff ? 0.f : theta[row];
    // Wave 0: wait until every tile sum of the row is visible, then the first
    // search over the tile sums.
    if (threadIdx.x < kWave) {
        const int lane = lane_id();
        bool failed = false;
        for (uint32_t b = 0; b < segs; b += kWave) {
            const uint32_t s = b + lane;
            if (s < segs) {
                uint64_t word;
                for (uint32_t spins = 0;; ++spins) {  // bounded: every tile has stored already
                    word = __hip_atomic_load(&rs[s], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    if (row_word(word) || spins >= kSpinLimit) break;
                    __builtin_amdgcn_s_sleep(1);
                }
                failed |= !row_word(word);
            }
        }
        if (__ballot(failed) && lane == 0)
            __hip_atomic_store(&hdr->error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        float excl = 0.f;
        const float thr = MODE == ToppMode::Weighted ? th * topp_total(rs, segs) : p;
        const int32_t t = topp_find_tile(rs, segs, thr, MODE == ToppMode::Weighted, &excl);
        if (lane == 0) {
            s_tile = t;
            s_excl = excl;
            s_thr = thr;
        }
    }
    __syncthreads();
    const int32_t t = s_tile;
    const float excl = s_excl, thr = s_thr;
    __syncthreads();  // s_tile / s_excl reused below
    int64_t found;    // the cutoff (cutoff / sample modes) or the weighted draw
    float at = excl;  // running sum at `found` (no tile: the row total)
    if (t < 0)
        found = len - 1;
    else
        found = topp_find<TileT, VEC, MODE == ToppMode::Weighted, MODE == ToppMode::Sample>(
            xr, len, (int64_t)t * TileT::kElems, excl, thr, len - 1, s_wtot, s_min, &s_val, at);
    if (MODE == ToppMode::Sample) {
        // second draw: among the kept indices 0..found, u = theta * C_found
        const float u = th * at;
        const uint32_t limit = t < 0 ? segs : (uint32_t)t + 1;
        if (threadIdx.x < kWave) {
            float e2 = 0.f;
            const int32_t t2 = topp_find_tile(rs, limit, u, true, &e2);
            if (lane_id() == 0) {
                s_tile = t2;
                s_excl = e2;
            }
        }
        __syncthreads();
        const int32_t t2 = s_tile;
        const float e2 = s_excl;
        int64_t j = found;
        float at2;
        if (t2 >= 0)
            j = topp_find<TileT, VEC, true, false>(xr, len, (int64_t)t2 * TileT::kElems, e2, u,
                                                    found, s_wtot, s_min, &s_val, at2);
        if (threadIdx.x == 0) {
            if (cutoff) cutoff[row] = (int32_t)found;
            token[row] = idx ? idx[row * len + j] : (int32_t)j;
        }
    } else if (threadIdx.x == 0) {
        (MODE == ToppMode::Cutoff ? cutoff : token)[row] = (int32_t)found;
    }
    // leave the row's sums and counter clear for the next call
    __syncthreads();
    for (uint32_t s = threadIdx.x; s < segs; s += TileT::kThreads)
        __hip_atomic_store(&rs[s], 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (threadIdx.x == 0)
        __hip_atomic_store(&arrivals[row], 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ---------------------------------------------------------------- weighted sampling, two kernels
//
// Rows of up to kWeightedMaxLen elements: no workgroup waits for another and
// none counts arrivals.  k_tile_sums stores the sum of every tile of every
// row (one read of the weights, all tiles at once); k_weighted_finish, one
// workgroup per row, adds the row's tile sums in tile order into the total
// W, finds the first tile whose inclusive sum exceeds theta * W, re-reads
// that one tile and finds the index in it (as k_topp does: should rounding
// leave the tile's running sums short of theta * W, its last index is
// taken).  The tile
// sums are plain fp32 values in the low halves of workspace words (the top
// bits clear, as the workspace invariant asks), written before they are read
// in every call.  This is k_topp's weighted mode with the row's last-arrival
// step replaced by a kernel boundary, which costs less than the per-row
// arrival atomics.
constexpr int64_t kWeightedMaxLen = int64_t(1) << 22;
static inline bool weighted_two_kernels(int64_t len) {
    return len > kRowTile && len <= kWeightedMaxLen;
}
static inline int64_t weighted_tile(int64_t len) { return len > 16384 ? 8192 : 4096; }

template <class TileT, bool VEC>
__global__ __launch_bounds__(TileT::kThreads) LS_OCCUPANCY4 void k_tile_sums(
    const float* x, int64_t len, uint32_t segs, uint64_t* sums) {
    __shared__ float s_wtot[TileT::WAVES];
    const int64_t row = blockIdx.x / segs;
    const uint32_t seg = blockIdx.x - (uint32_t)row * segs;
    float v[TileT::J][TileT::V];
    TileT::template load<VEC, true>(x + row * len, len, (int64_t)seg * TileT::kElems, v);
    float wofs;
    const float agg = TileT::combine_waves(wave_sum(TileT::lane_sum(v)), s_wtot, &wofs);
    if (threadIdx.x == 0) sums[blockIdx.x] = Bits<float>::to(agg);
}

template <class TileT, bool VEC>
__global__ __launch_bounds__(TileT::kThreads) LS_OCCUPANCY4 void k_weighted_finish(
    const float* w, const float* theta, int32_t* out, int64_t len, uint32_t segs,
    const uint64_t* sums) {
    __shared__ float s_wtot[TileT::WAVES];
    __shared__ int32_t s_min[TileT::WAVES];
    __shared__ float s_val;
    __shared__ int32_t s_tile;
    __shared__ float s_excl, s_thr;
    const int64_t row = blockIdx.x;
    const uint64_t* rs = sums + row * segs;
    if (threadIdx.x < kWave) {
        const float thr = theta[row] * topp_total(rs, segs);
        float excl = 0.f;
        const int32_t t = topp_find_tile(rs, segs, thr, true, &excl);
        if (lane_id() == 0) {
            s_tile = t;
            s_excl = excl;
            s_thr = thr;
        }
    }
    __syncthreads();
    const int32_t t = s_tile;
    int64_t found = len - 1;  // no tile exceeds theta * W (rounding): the last index
    if (t >= 0) {
        float at;
        found = topp_find<TileT, VEC, true, false>(w + row * len, len, (int64_t)t * TileT::kElems,
                                                   s_excl, s_thr, len - 1, s_wtot, s_min, &s_val,
                                                   at);
    }
    if (threadIdx.x == 0) out[row] = (int32_t)found;
}

// ---------------------------------------------------------------- top-p, early exit
//
// The cutoff for rows of 2 to kEarlyMaxSegs tiles of 4096 elements, reading
// little more of a row than the cutoff needs when the crossing lies in the
// row's head (as it does on sorted probabilities: the largest ones come
// first), with no workgroup ever waiting for another.  Two kernels:
//  * k_topp_head reads the first `heads` tiles of every row, all at once,
//    and stores for each tile its sum and the largest running sum inside it
//    (from the tile's start);
//  * k_topp_finish, one workgroup per row, scans those pairs in tile order:
//    tile t holds an index whose running sum reaches p exactly when
//    E_t + M_t >= p (E_t the sum of the tiles before it, M_t its largest
//    inner running sum; rounding is monotone, so this is exact for the
//    running sums as computed here), re-reads the first such tile (just
//    read) and finds the index; if the head holds none, it
//    walks the rest of the row itself, 8192 elements per step.
// A running sum is always taken as E + (tile-local inclusive sum), the same
// in both kernels, so the head's verdict and the search agree.  The result
// is the definition's on any input.  The head words are plain fp32 values in
// the low halves of 64-bit workspace words (the top bits clear, as the
// workspace invariant asks), written before they are read in every call.
constexpr int64_t kEarlyTile = 4096;
constexpr int64_t kEarlyMaxSegs = 256;  // rows up to 2^20 elements
// The finishing kernel re-reads a head tile with the head kernel's own tile
// geometry (the row tile of 4096: 4 waves of 4 chunks, or 8 waves of 2 for
// misaligned rows), so that its running sums are bit for bit the ones the
// head's words were taken from.
template <bool VEC>
using HeadTile = RowTile<float, RGeomS, VEC>;
template <bool VEC>
constexpr int kFinishThreads = HeadTile<VEC>::kThreads;

// Tiles of a row read by the head kernel: a quarter of the row, at least 8.
static inline uint32_t topp_heads(int64_t len) {
    const int64_t segs = (len + kEarlyTile - 1) / kEarlyTile;
    const int64_t q = (segs + 3) / 4 > 8 ? (segs + 3) / 4 : 8;
    return (uint32_t)(q < segs ? q : segs);
}

// Wavefront maximum with DPP (lanes outside the row / disabled read -inf).
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp_fmax(float v) {
    const float o = Bits<float>::from((uint32_t)__builtin_amdgcn_update_dpp(
        (int)0xff800000u, (int)Bits<float>::to(v), CTRL, ROW_MASK, 0xf, false));
    return o > v ? o : v;
}
__device__ __forceinline__ float wave_fmax(float v) {
    v = dpp_fmax<0x111, 0xf>(v);
    v = dpp_fmax<0x112, 0xf>(v);
    v = dpp_fmax<0x114, 0xf>(v);
    v = dpp_fmax<0x118, 0xf>(v);
    v = dpp_fmax<0x142, 0xa>(v);
    v = dpp_fmax<0x143, 0xc>(v);
    return lane_read(v, kWave - 1);
}

template <class TileT, bool VEC>
__global__ __launch_bounds__(TileT::kThreads) LS_OCCUPANCY4 void k_topp_head(
    const float* probs, int64_t len, uint32_t rows, uint32_t heads, uint64_t* words) {
    __shared__ float s_wtot[TileT::WAVES];
    __shared__ float s_wmax[TileT::WAVES];
    const uint32_t row32 = blockIdx.x % rows;  // tile t of every row before tile t + 1
    const uint32_t t = blockIdx.x / rows;
    const int64_t base = (int64_t)t * TileT::kElems;
    float v[TileT::J][TileT::V];
    // nontemporal loads (cold rows are not allocated in the Infinity Cache on
    // the way): 9.3 against 11.0 us per 128 x 131072 call with cached loads,
    // the finishing kernel's re-read of one tile per row included
    TileT::template load<VEC, true>(probs + (int64_t)row32 * len, len, base, v);
    float wofs;
    const float agg = TileT::combine_waves(TileT::template wave_scan<false>(v), s_wtot, &wofs);
    const int32_t valid = (int32_t)(len - base < TileT::kElems ? len - base : TileT::kElems);
    float mx = -__builtin_inff();
#pragma unroll
    for (int j = 0; j < TileT::J; ++j) {
        const int32_t off = (int32_t)TileT::lane_offset(j);
#pragma unroll
        for (int e = 0; e < TileT::V; ++e) {
            const float run = wofs + v[j][e];
            if (off + e < valid) mx = run > mx ? run : mx;
        }
    }
    mx = wave_fmax(mx);
    if (lane_id() == 0) s_wmax[threadIdx.x / kWave] = mx;
    __syncthreads();
    if (threadIdx.x == 0) {
        float m = s_wmax[0];
        for (int k = 1; k < TileT::WAVES; ++k) m = s_wmax[k] > m ? s_wmax[k] : m;
        uint64_t* w = words + ((size_t)row32 * heads + t) * 2;
        w[0] = Bits<float>::to(agg);
        w[1] = Bits<float>::to(m);
    }
}

// The whole workgroup: the first index i < valid of the tile in v whose
// running sum e + (wofs + v[i]) reaches p (STRICT: exceeds it), or INT_MAX;
// *val (when given) gets the running sum there.  Contains barriers.
template <class TileT, bool STRICT = false>
__device__ __forceinline__ int32_t topp_first_reach(const float (&v)[TileT::J][TileT::V],
                                                    float e, float wofs, int32_t valid, float p,
                                                    int32_t* s_min, float* s_val = nullptr,
                                                    float* val = nullptr) {
    int32_t cand = INT_MAX;
    float cand_val = 0.f;
#pragma unroll
    for (int j = TileT::J - 1; j >= 0; --j) {
        const int32_t off = (int32_t)TileT::lane_offset(j);
#pragma unroll
        for (int k = TileT::V - 1; k >= 0; --k) {
            const float run = e + (wofs + v[j][k]);
            if (off + k < valid && (STRICT ? run > p : run >= p)) {
                cand = off + k;
                cand_val = run;
            }
        }
    }
    const int32_t wm = wave_min(cand);
    if (lane_id() == 0) s_min[threadIdx.x / kWave] = wm;
    __syncthreads();
    int32_t m = INT_MAX;
    for (int k = 0; k < TileT::WAVES; ++k) m = s_min[k] < m ? s_min[k] : m;
    if (val) {
        if (m != INT_MAX && cand == m) *s_val = cand_val;  // exactly one lane
        __syncthreads();
        *val = *s_val;
    }
    __syncthreads();  // s_min / s_val are rewritten by the next call
    return m;
}

// Wave 0: the first head tile t in [from, limit) whose largest inner running
// sum E_t + M_t reaches p (STRICT: exceeds it), -1 if none; *e gets E_t (with
// none: the sum of the tiles [from, limit) added to carry).
__device__ __forceinline__ int32_t topp_head_tile(const uint64_t* hw, uint32_t from,
                                                  uint32_t limit, float carry, float p,
                                                  bool strict, float* e) {
    const int lane = lane_id();
    for (uint32_t b = from; b < limit; b += kWave) {
        const uint32_t t = b + lane;
        const float a = t < limit ? Bits<float>::from((uint32_t)hw[2 * t]) : 0.f;
        const float m = t < limit ? Bits<float>::from((uint32_t)hw[2 * t + 1]) : 0.f;
        const float sc = wave_incl_scan(a);
        const float ex = carry + wave_shr1(sc);  // E_t: the sum of the tiles before t
        const uint64_t hit = __ballot(t < limit && (strict ? ex + m > p : ex + m >= p));
        if (hit) {
            const int l = __builtin_ctzll(hit);
            *e = lane_read(ex, l);
            return (int32_t)(b + l);
        }
        carry = carry + lane_read(sc, kWave - 1);
    }
    *e = carry;
    return -1;
}

// The whole workgroup: the first index i <= lim of the row at xr whose
// running sum reaches thr (STRICT: exceeds it), -1 if none.  The head tiles'
// words pick the first head tile that holds one (E_t + M_t against thr), that
// tile is re-read with the head kernel's geometry and searched (the same sums,
// so the search finds what the words promised; should it not, the search goes
// on from the next head tile).
// With none in the head, the rest of the row is walked, 8192 elements per
// step.  *val gets the running sum at the index found, or (none) the sum of
// every element up to the end of the last tile searched.
template <bool VEC, bool STRICT>
__device__ int64_t topp_head_find(const float* xr, int64_t len, const uint64_t* hw, uint32_t heads,
                                  float thr, int64_t lim, float* val, int32_t* s_tile, float* s_e,
                                  float* s_wtot, int32_t* s_min, float* s_val) {
    using H = HeadTile<VEC>;  // one head tile, 4096, as the head kernel read it
    using B = Tile<float, float, 4, 2 * H::J, H::WAVES>;  // 8192 per step after the head
    static_assert(H::kElems == kEarlyTile && B::kElems == 2 * kEarlyTile, "head tile");
    const int64_t lim_tiles = lim / kEarlyTile + 1;  // head tiles holding indices <= lim
    const uint32_t limit = (uint32_t)(lim_tiles < (int64_t)heads ? lim_tiles : heads);
    float carry = 0.f;  // sum of the head tiles before `from`
    uint32_t from = 0;
    while (true) {
        if (threadIdx.x < kWave) {
            float e = 0.f;
            const int32_t t = topp_head_tile(hw, from, limit, carry, thr, STRICT, &e);
            if (lane_id() == 0) {
                *s_tile = t;
                *s_e = e;
            }
        }
        __syncthreads();
        const int32_t t = *s_tile;
        const float e = *s_e;
        __syncthreads();  // s_tile / s_e are rewritten by the next round
        if (t < 0) {
            carry = e;  // the sum of the head tiles searched
            break;
        }
        const int64_t base = (int64_t)t * H::kElems;
        float v[H::J][H::V];
        H::template load<VEC>(xr, len, base, v);
        float wofs;
        const float agg = H::combine_waves(H::template wave_scan<false>(v), s_wtot, &wofs);
        const int64_t end = (lim + 1 < len ? lim + 1 : len) - base;  // indices <= lim
        const int32_t valid = (int32_t)(end < H::kElems ? end : H::kElems);
        float at;
        const int32_t m = topp_first_reach<H, STRICT>(v, e, wofs, valid, thr, s_min, s_val, &at);
        if (m != INT_MAX) {
            *val = at;
            return base + m;
        }
        carry = e + agg;
        from = (uint32_t)t + 1;
        __syncthreads();  // s_wtot is rewritten by the next combine
    }
    for (int64_t base = (int64_t)limit * kEarlyTile; base <= lim && limit == heads;
         base += B::kElems) {
        float v[B::J][B::V];
        B::template load<VEC, true>(xr, len, base, v);
        float wofs;
        const float agg = B::combine_waves(B::template wave_scan<false>(v), s_wtot, &wofs);
        const int64_t end = (lim + 1 < len ? lim + 1 : len) - base;
        const int32_t valid = (int32_t)(end < B::kElems ? end : B::kElems);
        float at;
        const int32_t m = topp_first_reach<B, STRICT>(v, carry, wofs, valid, thr, s_min, s_val, &at);
        if (m != INT_MAX) {
            *val = at;
            return base + m;
        }
        carry = carry + agg;
        __syncthreads();  // s_wtot is rewritten by the next combine
    }
    *val = carry;
    return -1;
}

// The cutoff k (len - 1 when no running sum reaches p); SAMPLE: the top-p
// draw on the sorted rows as well -- with C the running sum at k, the first
// index j <= k whose running sum exceeds theta * C (j = k when rounding
// leaves none), found the same way; the token is idx[j] (idx null: j
// itself), and the cutoff is stored only when asked for.
template <bool VEC, bool SAMPLE>
__global__ __launch_bounds__(kFinishThreads<VEC>) LS_OCCUPANCY4 void k_topp_finish(
    const float* probs, int32_t* cutoff, int64_t len, uint32_t heads, float p,
    const uint64_t* words, const int32_t* idx, const float* theta, int32_t* token) {
    __shared__ int32_t s_tile;
    __shared__ float s_e;
    __shared__ float s_wtot[kFinishThreads<VEC> / kWave];
    __shared__ int32_t s_min[kFinishThreads<VEC> / kWave];
    __shared__ float s_val;

    const uint32_t row32 = blockIdx.x;
    const float* xr = probs + (int64_t)row32 * len;
    const uint64_t* hw = words + (size_t)row32 * heads * 2;
    float c;  // the running sum at k (none reached: the row total)
    int64_t k = topp_head_find<VEC, false>(xr, len, hw, heads, p, len - 1, &c, &s_tile, &s_e,
                                           s_wtot, s_min, &s_val);
    if (k < 0) k = len - 1;
    if (!SAMPLE) {
        if (threadIdx.x == 0) cutoff[row32] = (int32_t)k;
        return;
    }
    __syncthreads();
    float at;
    int64_t j = topp_head_find<VEC, true>(xr, len, hw, heads, theta[row32] * c, k, &at, &s_tile,
                                          &s_e, s_wtot, s_min, &s_val);
    if (j < 0) j = k;
    if (threadIdx.x == 0) {
        if (cutoff) cutoff[row32] = (int32_t)k;
        token[row32] = idx ? idx[(int64_t)row32 * len + j] : (int32_t)j;
    }
}

__global__ void k_fill_i32(int32_t* p, int64_t count, int32_t value) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += stride) p[i] = value;
}

// ---------------------------------------------------------------- short rows

template <class T, bool EXCL, bool VEC, bool TOPP>
__global__ __launch_bounds__(256) void k_rows_wave(const T* x, T* y, int64_t rows, int64_t len,
                                                   float p, int32_t* cutoff) {
    constexpr int V = 4;
    const int lane = lane_id();
    const int64_t nw = (int64_t)gridDim.x * (blockDim.x / kWave);
    for (int64_t r = (int64_t)blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave; r < rows;
         r += nw) {
        const T* xr = x + r * len;
        T carry = T(0);
        int32_t found = -1;
        for (int64_t c = 0; c < len; c += kWave * V) {
            const int64_t off = c + (int64_t)lane * V;
            T v[V];
            if (VEC && c + kWave * V <= len) {
                load_vec<T, T, V>(xr + off, v);
            } else {
#pragma unroll
                for (int e = 0; e < V; ++e) v[e] = off + e < len ? xr[off + e] : T(0);
            }
#pragma unroll
            for (int e = 1; e < V; ++e) v[e] = v[e - 1] + v[e];
            const T inc = wave_incl_scan(v[V - 1]);
            const T lb = carry + wave_shr1(inc);
            if constexpr (!TOPP) {
                T o[V];
#pragma unroll
                for (int e = 0; e < V; ++e) o[e] = EXCL ? (e == 0 ? lb : lb + v[e - 1]) : lb + v[e];
                T* yr = y + r * len;
                if (VEC && c + kWave * V <= len) {
                    store_vec<T, V>(yr + off, o);
                } else {
#pragma unroll
                    for (int e = 0; e < V; ++e)
                        if (off + e < len) yr[off + e] = o[e];
                }
            } else {
                int32_t hit = INT_MAX;
#pragma unroll
                for (int e = V - 1; e >= 0; --e)
                    if (off + e < len && lb + v[e] >= p) hit = (int32_t)(off + e);
                const uint64_t m = __ballot(hit != INT_MAX);
                if (m) {  // lanes are in index order: the lowest hitting lane has the first hit
                    found = __builtin_amdgcn_readlane(hit, __builtin_ctzll(m));
                    break;
                }
            }
            carry = carry + lane_read(inc, kWave - 1);
        }
        if (TOPP && lane == 0) cutoff[r] = found >= 0 ? found : (int32_t)(len - 1);
    }
}

// ---------------------------------------------------------------- launchers

// Long rows: header | one status word (row scan) or tile sum (top-p) per
// smallest-geometry segment | one top-p arrival counter per row.
static size_t topp_arrivals_offset(int64_t rows, int64_t len) {
    return kWsHeader + (size_t)rows * (size_t)row_segments(len) * sizeof(uint64_t);
}
size_t topp_ws_bytes(int64_t rows, int64_t len) {
    return topp_arrivals_offset(rows, len) + (size_t)rows * sizeof(uint64_t);
}
// Weighted sampling: the top-p layout, or one tile sum per row tile of the
// two-kernel path.
size_t weighted_ws_bytes(int64_t rows, int64_t len) {
    const size_t a = topp_ws_bytes(rows, len);
    if (!weighted_two_kernels(len)) return a;
    const int64_t t = weighted_tile(len);
    const size_t b = kWsHeader + (size_t)rows * (size_t)((len + t - 1) / t) * sizeof(uint64_t);
    return a > b ? a : b;
}
static bool topp_early(int64_t len);
static size_t topp_early_ws_bytes(int64_t rows, int64_t len);
size_t scan_rows_ws_bytes(int64_t rows, int64_t len) {
    // short rows (one wavefront per row) need no workspace beyond the header
    if (!long_rows(len)) return kWsHeader;
    const size_t a = topp_ws_bytes(rows, len);
    const size_t b = topp_early(len) ? topp_early_ws_bytes(rows, len) : 0;
    return a > b ? a : b;
}

static bool aligned16(const void* p) { return ((uintptr_t)p % 16) == 0; }

static unsigned wave_grid(int64_t rows) {
    const int64_t blocks = (rows + 3) / 4;
    return (unsigned)(blocks < 65536 ? blocks : 65536);
}

template <class T, class G>
static void rows_long(bool exclusive, bool vec, const T* x, T* y, int64_t rows, int64_t len,
                      void* ws, size_t ws_bytes, hipStream_t stream) {
    using TV = RowTile<T, G, true>;
    using TU = RowTile<T, G, false>;
    static_assert(TV::kElems == TU::kElems, "one tile size per geometry");
    const uint32_t segs = (uint32_t)((len + TV::kElems - 1) / TV::kElems);
    const uint32_t nt = (uint32_t)(rows * segs);
    WsHeader* hdr = reinterpret_cast<WsHeader*>(ws);
    uint64_t* status = reinterpret_cast<uint64_t*>(reinterpret_cast<char*>(ws) + kWsHeader);
    const int64_t status_words = (int64_t)((ws_bytes - kWsHeader) / sizeof(uint64_t));
    auto k = exclusive ? (vec ? k_rows_lookback<TV, true, true> : k_rows_lookback<TU, true, false>)
                       : (vec ? k_rows_lookback<TV, false, true> : k_rows_lookback<TU, false, false>);
    const unsigned threads = vec ? TV::kThreads : TU::kThreads;
    hipLaunchKernelGGL(k, dim3(nt), dim3(threads), 0, stream, x, y, len, segs, nt, hdr, status,
                       status_words);
}

template <class G, ToppMode MODE>
static void topp_long(bool vec, const float* probs, const int32_t* idx, const float* theta,
                      int32_t* cutoff, int32_t* token, int64_t rows, int64_t len, float p,
                      void* ws, hipStream_t stream) {
    using TV = RowTile<float, G, true>;
    using TU = RowTile<float, G, false>;
    const uint32_t segs = (uint32_t)((len + TV::kElems - 1) / TV::kElems);
    const uint32_t nt = (uint32_t)(rows * segs);
    const unsigned threads = vec ? TV::kThreads : TU::kThreads;
    uint64_t* sums = reinterpret_cast<uint64_t*>(reinterpret_cast<char*>(ws) + kWsHeader);
    uint64_t* arrivals = reinterpret_cast<uint64_t*>(reinterpret_cast<char*>(ws) +
                                                     topp_arrivals_offset(rows, len));
    auto k = vec ? k_topp<TV, true, MODE> : k_topp<TU, false, MODE>;
    hipLaunchKernelGGL(k, dim3(nt), dim3(threads), 0, stream, probs, idx, theta, cutoff, token,
                       len, segs, p, reinterpret_cast<WsHeader*>(ws), sums, arrivals);
}

// Rows of 2 to kEarlyMaxSegs tiles of 4096 take the early-exit cutoff kernels.
static bool topp_early(int64_t len) {
    return len > kEarlyTile && (len + kEarlyTile - 1) / kEarlyTile <= kEarlyMaxSegs;
}
static size_t topp_early_ws_bytes(int64_t rows, int64_t len) {
    return kWsHeader + (size_t)rows * topp_heads(len) * 2 * sizeof(uint64_t);
}

static void topp_cutoff_early(bool vec, const float* probs, int32_t* cutoff, int64_t rows,
                              int64_t len, float p, void* ws, hipStream_t stream) {
    using TV = RowTile<float, RGeomS, true>;
    using TU = RowTile<float, RGeomS, false>;
    static_assert(TV::kElems == kEarlyTile && TU::kElems == kEarlyTile, "early-exit tile");
    const uint32_t heads = topp_heads(len);
    uint64_t* words = reinterpret_cast<uint64_t*>(reinterpret_cast<char*>(ws) + kWsHeader);
    auto kh = vec ? k_topp_head<TV, true> : k_topp_head<TU, false>;
    hipLaunchKernelGGL(kh, dim3((unsigned)(rows * heads)), dim3(vec ? TV::kThreads : TU::kThreads),
                       0, stream, probs, len, (uint32_t)rows, heads, words);
    auto kf = vec ? k_topp_finish<true, false> : k_topp_finish<false, false>;
    hipLaunchKernelGGL(kf, dim3((unsigned)rows),
                       dim3(vec ? kFinishThreads<true> : kFinishThreads<false>), 0,
                       stream, probs, cutoff,
                       len, heads, p, words, nullptr, nullptr, nullptr);
}

// The top-p draw on sorted rows by the same two kernels (rows as topp_early).
static void topp_sample_early(bool vec, const float* sorted, const int32_t* idx,
                              const float* theta, int32_t* cutoff, int32_t* token, int64_t rows,
                              int64_t len, float p, void* ws, hipStream_t stream) {
    using TV = RowTile<float, RGeomS, true>;
    using TU = RowTile<float, RGeomS, false>;
    const uint32_t heads = topp_heads(len);
    uint64_t* words = reinterpret_cast<uint64_t*>(reinterpret_cast<char*>(ws) + kWsHeader);
    auto kh = vec ? k_topp_head<TV, true> : k_topp_head<TU, false>;
    hipLaunchKernelGGL(kh, dim3((unsigned)(rows * heads)), dim3(vec ? TV::kThreads : TU::kThreads),
                       0, stream, sorted, len, (uint32_t)rows, heads, words);
    auto kf = vec ? k_topp_finish<true, true> : k_topp_finish<false, true>;
    hipLaunchKernelGGL(kf, dim3((unsigned)rows),
                       dim3(vec ? kFinishThreads<true> : kFinishThreads<false>), 0,
                       stream, sorted, cutoff,
                       len, heads, p, words, idx, theta, token);
}

template <ToppMode MODE>
static void topp_any(bool vec, const float* probs, const int32_t* idx, const float* theta,
                     int32_t* cutoff, int32_t* token, int64_t rows, int64_t len, float p,
                     void* ws, hipStream_t stream) {
    if (MODE == ToppMode::Cutoff && topp_early(len)) {
        topp_cutoff_early(vec, probs, cutoff, rows, len, p, ws, stream);
        return;
    }
    if (MODE == ToppMode::Sample && topp_early(len)) {
        topp_sample_early(vec, probs, idx, theta, cutoff, token, rows, len, p, ws, stream);
        return;
    }
    const int64_t t = row_tile(len);
    if (t == 32768)
        topp_long<RGeomL, MODE>(vec, probs, idx, theta, cutoff, token, rows, len, p, ws, stream);
    else if (t == 8192)
        topp_long<RGeomM, MODE>(vec, probs, idx, theta, cutoff, token, rows, len, p, ws, stream);
    else
        topp_long<RGeomS, MODE>(vec, probs, idx, theta, cutoff, token, rows, len, p, ws, stream);
}

template <class T, bool TOPP>
static hipError_t rows_typed(bool exclusive, const T* x, T* y, int64_t rows, int64_t len, float p,
                             int32_t* cutoff, void* ws, size_t ws_bytes, hipStream_t stream) {
    if (rows == 0) return hipSuccess;
    if (len == 0) {
        if (TOPP)
            hipLaunchKernelGGL(k_fill_i32, dim3(wave_grid(rows)), dim3(256), 0, stream, cutoff,
                               rows, (int32_t)-1);
        return hipGetLastError();
    }
    const bool vec = (len % 4 == 0) && aligned16(x) && (TOPP || aligned16(y));
    if (!TOPP && !long_rows(len) && len > kRowsTileMin) {
        using TV = RowTile<T, RGeomS, true>;
        using TU = RowTile<T, RGeomS, false>;
        static_assert(TV::kElems == kRowTile && TU::kElems == kRowTile, "one tile per row");
        auto k = exclusive ? (vec ? k_rows_tile<TV, true, true> : k_rows_tile<TU, true, false>)
                           : (vec ? k_rows_tile<TV, false, true> : k_rows_tile<TU, false, false>);
        hipLaunchKernelGGL(k, dim3((unsigned)rows), dim3(vec ? TV::kThreads : TU::kThreads), 0,
                           stream, x, y, len);
        return hipGetLastError();
    }
    if (!long_rows(len)) {
        const dim3 grid(wave_grid(rows)), block(256);
        auto k = exclusive ? (vec ? k_rows_wave<T, true, true, TOPP> : k_rows_wave<T, true, false, TOPP>)
                           : (vec ? k_rows_wave<T, false, true, TOPP> : k_rows_wave<T, false, false, TOPP>);
        hipLaunchKernelGGL(k, grid, block, 0, stream, x, y, rows, len, p, cutoff);
        return hipGetLastError();
    }
    const int64_t t = row_tile(len);
    if constexpr (TOPP) {
        topp_any<ToppMode::Cutoff>(vec, x, nullptr, nullptr, cutoff, nullptr, rows, len, p, ws,
                                   stream);
    } else {
        if (t == 32768) rows_long<T, RGeomL>(exclusive, vec, x, y, rows, len, ws, ws_bytes, stream);
        else if (t == 8192) rows_long<T, RGeomM>(exclusive, vec, x, y, rows, len, ws, ws_bytes, stream);
        else rows_long<T, RGeomS>(exclusive, vec, x, y, rows, len, ws, ws_bytes, stream);
    }
    return hipGetLastError();
}

hipError_t launch_scan_rows(Kind kind, bool exclusive, const void* x, void* y, int64_t rows,
                            int64_t len, void* ws, size_t ws_bytes, hipStream_t stream) {
    switch (kind) {
        case Kind::I32:
            return rows_typed<uint32_t, false>(exclusive, (const uint32_t*)x, (uint32_t*)y, rows,
                                               len, 0.f, nullptr, ws, ws_bytes, stream);
        case Kind::F32:
            return rows_typed<float, false>(exclusive, (const float*)x, (float*)y, rows, len, 0.f,
                                            nullptr, ws, ws_bytes, stream);
        default:
            return hipErrorInvalidValue;
    }
}

hipError_t launch_topp_cutoff(const float* probs, int32_t* cutoff, int64_t rows, int64_t len,
                              float p, void* ws, size_t ws_bytes, hipStream_t stream) {
    return rows_typed<float, true>(false, probs, nullptr, rows, len, p, cutoff, ws, ws_bytes,
                                   stream);
}

template <class G>
static void weighted_two(bool vec, const float* w, const float* theta, int32_t* out, int64_t rows,
                         int64_t len, void* ws, hipStream_t stream) {
    using TV = RowTile<float, G, true>;
    using TU = RowTile<float, G, false>;
    static_assert(TV::kElems == TU::kElems, "one tile size per geometry");
    const uint32_t segs = (uint32_t)((len + TV::kElems - 1) / TV::kElems);
    const unsigned threads = vec ? TV::kThreads : TU::kThreads;
    uint64_t* sums = reinterpret_cast<uint64_t*>(reinterpret_cast<char*>(ws) + kWsHeader);
    hipLaunchKernelGGL((vec ? k_tile_sums<TV, true> : k_tile_sums<TU, false>),
                       dim3((unsigned)(rows * segs)), dim3(threads), 0, stream, w, len, segs, sums);
    hipLaunchKernelGGL((vec ? k_weighted_finish<TV, true> : k_weighted_finish<TU, false>),
                       dim3((unsigned)rows), dim3(threads), 0, stream, w, theta, out, len, segs,
                       (const uint64_t*)sums);
}

// Appendix "Weighted Sampling", per row (any length; workspace
// weighted_ws_bytes(rows, len)).
hipError_t launch_weighted_sample(const float* w, const float* theta, int32_t* out, int64_t rows,
                                  int64_t len, void* ws, hipStream_t stream) {
    if (rows == 0) return hipSuccess;
    if (len == 0) {
        hipLaunchKernelGGL(k_fill_i32, dim3(wave_grid(rows)), dim3(256), 0, stream, out, rows,
                           (int32_t)-1);
        return hipGetLastError();
    }
    const bool vec = (len % 4 == 0) && aligned16(w);
    if (weighted_two_kernels(len)) {
        if (weighted_tile(len) == 8192)
            weighted_two<RGeomM>(vec, w, theta, out, rows, len, ws, stream);
        else
            weighted_two<RGeomS>(vec, w, theta, out, rows, len, ws, stream);
    } else {
        topp_any<ToppMode::Weighted>(vec, w, nullptr, theta, nullptr, out, rows, len, 0.f, ws,
                                     stream);
    }
    return hipGetLastError();
}

// The top-p draw on rows already sorted in descending order: cutoff k, then
// the draw among 0..k, reported through idx (workspace topp_ws_bytes).
hipError_t launch_topp_draw_sorted(const float* sorted, const int32_t* idx, const float* theta,
                                   float p, int32_t* token, int32_t* cutoff, int64_t rows,
                                   int64_t len, void* ws, hipStream_t stream) {
    if (rows == 0) return hipSuccess;
    if (len == 0) {
        hipLaunchKernelGGL(k_fill_i32, dim3(wave_grid(rows)), dim3(256), 0, stream, token, rows,
                           (int32_t)-1);
        if (cutoff)
            hipLaunchKernelGGL(k_fill_i32, dim3(wave_grid(rows)), dim3(256), 0, stream, cutoff,
                               rows, (int32_t)-1);
        return hipGetLastError();
    }
    const bool vec = (len % 4 == 0) && aligned16(sorted);
    topp_any<ToppMode::Sample>(vec, sorted, idx, theta, cutoff, token, rows, len, p, ws, stream);
    return hipGetLastError();
}

// The top-p sampler on unsorted rows (Section 5 "Top-p or Nucleus Sampling"):
// a stable descending radix sort of each row, keeping source indices, then
// the cutoff and the draw on the sorted row.  Workspace: the sort's and the
// draw's common head.  Scratch (caller memory with no invariant, since it
// ends up holding sort codes): four rows x len arrays -- sorted keys, their
// source indices, and the sort's two ping-pong buffers.
static size_t align256(size_t b) { return (b + 255) / 256 * 256; }
size_t topp_sample_ws_bytes(int64_t rows, int64_t len) {
    const size_t a = radix_rows_ws_bytes(rows, len), b = scan_rows_ws_bytes(rows, len);
    return a > b ? a : b;
}
size_t topp_sample_scratch_bytes(int64_t rows, int64_t len) {
    return 4 * align256((size_t)rows * (size_t)len * 4);
}
hipError_t launch_topp_sample(const float* probs, const float* theta, float p, int32_t* token,
                              int32_t* cutoff, int64_t rows, int64_t len, void* scratch, void* ws,
                              hipStream_t stream) {
    if (rows == 0) return hipSuccess;
    if (len == 0)
        return launch_topp_draw_sorted(probs, nullptr, theta, p, token, cutoff, rows, len, ws,
                                       stream);
    const size_t mb = align256((size_t)rows * (size_t)len * 4);
    char* base = reinterpret_cast<char*>(scratch);
    float* sorted = reinterpret_cast<float*>(base);
    int32_t* perm = reinterpret_cast<int32_t*>(base + mb);
    float* keys_tmp = reinterpret_cast<float*>(base + 2 * mb);
    int32_t* perm_tmp = reinterpret_cast<int32_t*>(base + 3 * mb);
    const hipError_t e =
        launch_radix_sort_typed(KeyType::F32, true, probs, sorted, nullptr, perm, keys_tmp,
                                perm_tmp, rows, len, ws, topp_sample_ws_bytes(rows, len), stream);
    if (e != hipSuccess) return e;
    return launch_topp_draw_sorted(sorted, perm, theta, p, token, cutoff, rows, len, ws, stream);
}

}  // namespace ls
