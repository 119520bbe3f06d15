// topk.hip -- top-k of every row of a row-major rows x len fp32 matrix
// (Section 5 "Top-k": selection, a partial quicksort, on stable splits).
//
// Quickselect narrows the candidates around one pivot per level.  Here the
// pivots come from the key bits: four rounds of an 8-bit digit histogram
// over the row's candidates find, per row, the key T of the k-th largest
// element and how many of the elements equal to T belong to the top k (kk);
// each round keeps one digit bucket as the candidates, as a quickselect
// level keeps one side of its pivot.  Then one stable split of the row takes
// every element above T and the first kk equal to T, in index order, and a
// stable sort of those k elements puts them in order.  Keys are the IEEE 754
// totalOrder codes of the values, complemented when the k smallest are
// asked for, so that the selection always takes the k largest keys.
//
// Rows of up to 2^17 elements with k <= 8192 take a shorter route after the
// first round: every key whose top digit is at least the chosen bucket's is
// a candidate, and when a row has at most 16384 of them they are gathered
// and one workgroup per row sorts them in LDS and keeps the first k (two
// reads of each row instead of five); a row with more candidates is
// finished by that workgroup alone (the three further rounds and the
// selection over its row).  That route's first round is two kernels: the
// tiles store their counts, then one workgroup per row adds them.  With
// k <= 256 the candidates come from one read instead: each tile keeps its
// keys at or above its own k-th key's top 16 bits (k_topk_tilesel).
//
// No workgroup waits for another during the histogram rounds: each tile
// writes its 256 digit counts to its own slots, and (on the longer route)
// the row's last tile to arrive (the per-row arrival counter of the row
// kernels) adds them and picks the bucket.  The split is a two-chain decoupled look-back (elements
// above T, elements equal to T), so the output keeps index order.
#include <limits.h>

#include <type_traits>

#include "launch.hpp"
#include "rowtile.hpp"

namespace ls {

constexpr int kTopkDigits = 256;

// Key of a value: its totalOrder code (an unsigned order on all bit
// patterns, the radix sort's encoding), complemented for the k smallest.
__device__ __forceinline__ uint32_t topk_key(uint32_t bits, bool largest) {
    const uint32_t c = bits ^ ((bits >> 31) ? 0xFFFFFFFFu : 0x80000000u);
    return largest ? c : ~c;
}

// Whether a key lies in the bucket the earlier rounds kept (its top 8R bits
// equal the row's prefix).
template <int R>
__device__ __forceinline__ bool topk_in_bucket(uint32_t key, uint32_t prefix) {
    if constexpr (R == 0)
        return true;
    else
        return (key >> (32 - 8 * R)) == prefix;
}

// Round R (0..3): per tile, the counts of digit (key >> (24 - 8R)) & 255 over
// the keys in the row's bucket; the row's last tile adds the tiles' counts,
// takes the digit d whose bucket holds the kk-th largest key -- the keys with
// a larger digit number fewer than kk, with digit >= d at least kk -- and
// leaves prefix = prefix * 256 + d and kk minus the keys above the bucket in
// the row's state (two 64-bit words per row; round 0 starts from prefix 0,
// kk = k).
template <class TileT, bool VEC, int R>
__global__ __launch_bounds__(TileT::kThreads) LS_OCCUPANCY4 void k_topk_hist(
    const uint32_t* x, int64_t len, uint32_t segs, uint32_t k, bool largest, uint32_t* hist,
    uint64_t* state, uint64_t* arrivals) {
    constexpr int kWaves = TileT::WAVES;
    // Several histograms per wave (picked by lane), so that equal digits in
    // one instruction collide at most 64 / kSub ways: the top digits of
    // probability-like data take a handful of values.
    constexpr int kSub = kWaves <= 8 ? 4 : 2;
    static_assert(TileT::kThreads >= kTopkDigits, "one thread per digit");
    __shared__ uint32_t s_h[kWaves * kSub][kTopkDigits];
    __shared__ uint32_t s_part[kTopkDigits / kWave];
    __shared__ uint32_t s_last;

    for (int i = threadIdx.x; i < kWaves * kSub * kTopkDigits; i += TileT::kThreads)
        (&s_h[0][0])[i] = 0;
    const uint32_t row32 = blockIdx.x / segs;
    const uint32_t seg = blockIdx.x - row32 * segs;
    const int64_t row = row32;
    const int64_t base = (int64_t)seg * TileT::kElems;
    const uint32_t prefix = R == 0 ? 0u : (uint32_t)state[2 * row];
    uint32_t v[TileT::J][TileT::V];
    TileT::template load<VEC>(x + row * len, len, base, v);
    __syncthreads();  // histograms cleared

    const int w = threadIdx.x / kWave;
    uint32_t* h = s_h[w * kSub + (lane_id() & (kSub - 1))];
    const int32_t valid = (int32_t)(len - base < TileT::kElems ? len - base : TileT::kElems);
    constexpr int kShift = 24 - 8 * R;
#pragma unroll
    for (int j = 0; j < TileT::J; ++j) {
        const int32_t off = (int32_t)TileT::lane_offset(j);
#pragma unroll
        for (int e = 0; e < TileT::V; ++e) {
            const uint32_t key = topk_key(v[j][e], largest);
            if (off + e < valid && topk_in_bucket<R>(key, prefix))
                atomicAdd(&h[(key >> kShift) & 255u], 1u);
        }
    }
    __syncthreads();
    if (threadIdx.x < kTopkDigits) {
        uint32_t t = 0;
#pragma unroll
        for (int q = 0; q < kWaves * kSub; ++q) t += s_h[q][threadIdx.x];
        // agent scope: written through, so the row's last tile reads it
        __hip_atomic_store(&hist[((int64_t)row32 * segs + seg) * kTopkDigits + threadIdx.x], t,
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __builtin_amdgcn_s_waitcnt(0);  // every count acknowledged before the tile arrives
    __syncthreads();
    if (threadIdx.x == 0) s_last = row_arrive(&arrivals[row]) == segs - 1;
    __syncthreads();
    if (!s_last) return;  // uniform over the workgroup

    // The row's last tile.  Thread t takes digit 255 - t, so an inclusive scan
    // over t counts the keys with a digit >= its own.
    const uint32_t* rh = hist + (int64_t)row32 * segs * kTopkDigits;
    const int t = threadIdx.x;
    uint32_t cnt = 0;
    if (t < kTopkDigits) {
        const int d = kTopkDigits - 1 - t;
        for (uint32_t s = 0; s < segs; ++s)
            cnt += __hip_atomic_load(&rh[(int64_t)s * kTopkDigits + d], __ATOMIC_RELAXED,
                                     __HIP_MEMORY_SCOPE_AGENT);
    }
    const uint32_t inc = wave_incl_scan(cnt);
    if (t < kTopkDigits && lane_id() == kWave - 1) s_part[w] = inc;
    __syncthreads();
    if (t < kTopkDigits) {
        uint32_t before = 0;
        for (int q = 0; q < w; ++q) before += s_part[q];
        const uint32_t at_least = before + inc;  // keys with digit >= 255 - t
        const uint32_t above = at_least - cnt;   // keys with digit > 255 - t
        const uint32_t kk = R == 0 ? k : (uint32_t)state[2 * row + 1];
        if (above < kk && kk <= at_least) {  // exactly one thread
            state[2 * row] = (uint64_t)((prefix << 8) | (uint32_t)(kTopkDigits - 1 - t));
            state[2 * row + 1] = (uint64_t)(kk - above);
        }
    }
    if (t == 0)
        __hip_atomic_store(&arrivals[row], 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The split (Section 5 "Split", stable, with indices): with T = the row's
// final prefix and kk its count, every key above T goes to position
// (keys above T before it) and every key equal to T to position
// (k - kk) + (keys equal to T before it) if that count is below kk.  The two
// counts before a tile come from two decoupled look-back chains over the
// row's tiles; inside the tile they are the exclusive tile scan of flags
// packed as (above << 16) | equal (at most 32768 each per tile).  Values are
// re-read for the few kept elements.
template <class TileT, bool VEC>
__global__ __launch_bounds__(TileT::kThreads) LS_OCCUPANCY4 void k_topk_select(
    const uint32_t* x, int64_t len, uint32_t segs, uint32_t ntiles, uint32_t k, bool largest,
    const uint64_t* state, uint32_t* sel_vals, int32_t* sel_idx, WsHeader* hdr, uint64_t* status,
    int64_t status_words) {
    static_assert(TileT::J * TileT::V <= 64, "per-lane flag masks are 64-bit");
    static_assert(TileT::kElems < 65536, "packed 16-bit tile counts");
    __shared__ Ticket s_ticket;
    __shared__ uint32_t s_wtot[TileT::WAVES];
    __shared__ uint32_t s_above, s_equal;

    if (threadIdx.x == 0) s_ticket = take_ticket(hdr, ntiles);
    __syncthreads();
    const uint32_t tile32 = (uint32_t)__builtin_amdgcn_readfirstlane(s_ticket.tile);
    const uint32_t epoch = (uint32_t)__builtin_amdgcn_readfirstlane(s_ticket.epoch);
    if (tile32 >= ntiles) {  // only with a workspace that was never zero-filled
        if (threadIdx.x == 0)
            __hip_atomic_store(&hdr->error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return;
    }
    const uint32_t row32 = tile32 / segs;
    const int64_t row = row32;
    const int64_t base = (int64_t)(tile32 - row32 * segs) * TileT::kElems;
    const uint32_t thr = (uint32_t)state[2 * row];
    const uint32_t kk = (uint32_t)state[2 * row + 1];
    const uint32_t n_above = k - kk;

    uint32_t v[TileT::J][TileT::V];
    TileT::template load<VEC>(x + row * len, len, base, v);
    const int32_t valid = (int32_t)(len - base < TileT::kElems ? len - base : TileT::kElems);
    uint64_t above_m = 0, equal_m = 0;
#pragma unroll
    for (int j = 0; j < TileT::J; ++j) {
        const int32_t off = (int32_t)TileT::lane_offset(j);
#pragma unroll
        for (int e = 0; e < TileT::V; ++e) {
            const uint32_t key = topk_key(v[j][e], largest);
            const bool in = off + e < valid;
            const bool a = in && key > thr, q = in && key == thr;
            above_m |= (uint64_t)a << (j * TileT::V + e);
            equal_m |= (uint64_t)q << (j * TileT::V + e);
            v[j][e] = (a ? 0x10000u : 0u) | (q ? 1u : 0u);
        }
    }
    uint32_t wofs;
    const uint32_t agg =
        TileT::combine_waves(TileT::template wave_scan<true>(v), s_wtot, &wofs);
    if (threadIdx.x < kWave) {
        const uint32_t first = row32 * segs;
        const uint32_t a = lookback<uint32_t>(status, tile32, first, agg >> 16, 0u, epoch, hdr);
        const uint32_t q =
            lookback<uint32_t>(status + ntiles, tile32, first, agg & 0xFFFFu, 0u, epoch, hdr);
        if (threadIdx.x == 0) {
            s_above = a;
            s_equal = q;
            finish_epoch(hdr, epoch, ntiles, status, status_words);
        }
    }
    __syncthreads();
    if ((above_m | equal_m) == 0) return;
    const uint32_t a0 = s_above + (wofs >> 16), q0 = s_equal + (wofs & 0xFFFFu);
    const uint32_t* xr = x + row * len;
    uint32_t* ov = sel_vals + row * k;
    int32_t* oi = sel_idx + row * k;
#pragma unroll
    for (int j = 0; j < TileT::J; ++j) {
        const int64_t off = TileT::offset(base, j);
#pragma unroll
        for (int e = 0; e < TileT::V; ++e) {
            const int bit = j * TileT::V + e;
            uint32_t pos = UINT_MAX;
            if ((above_m >> bit) & 1u) {
                pos = a0 + (v[j][e] >> 16);
                if (pos >= n_above) pos = UINT_MAX;  // cannot happen; guards the output
            } else if ((equal_m >> bit) & 1u) {
                const uint32_t r = q0 + (v[j][e] & 0xFFFFu);
                if (r < kk) pos = n_above + r;
            }
            if (pos != UINT_MAX) {
                ov[pos] = xr[off + e];
                oi[pos] = (int32_t)(off + e);
            }
        }
    }
}

// Sorts s[0, npow) (a power of two) in descending order by a bitonic
// network, `nthreads` threads of the workgroup taking the pairs.
__device__ __forceinline__ void bitonic_desc(uint64_t* s, uint32_t npow, uint32_t nthreads) {
    for (uint32_t size = 2; size <= npow; size <<= 1) {
        for (uint32_t stride = size >> 1; stride > 0; stride >>= 1) {
            for (uint32_t t = threadIdx.x; t < npow / 2; t += nthreads) {
                const uint32_t i = 2 * t - (t & (stride - 1));  // lower end of pair t
                const uint32_t j = i + stride;
                const uint64_t a = s[i], b = s[j];
                // blocks of `size` alternate direction; the last merge is descending
                if ((a < b) == ((i & size) == 0)) {
                    s[i] = b;
                    s[j] = a;
                }
            }
            __syncthreads();
        }
    }
}

// The kept elements in order, for k <= kTopkSortMax: one workgroup per row
// sorts the row's k (key, index) pairs in LDS by a bitonic network on the
// 64-bit composite key << 32 | ~index in descending order -- larger keys
// first, equal keys by increasing index, so the order is the stable one and
// unique -- padded with zeros (below every composite, whose low word is at
// least 2^31) to a power of two.  Values are decoded from the keys.
constexpr int kTopkSortMax = 8192;
constexpr int kTopkSortThreads = 512;
__global__ __launch_bounds__(kTopkSortThreads) void k_topk_sort(
    const uint32_t* sel_vals, const int32_t* sel_idx, uint32_t* values, int32_t* indices,
    uint32_t k, uint32_t npow, bool largest) {
    __shared__ uint64_t s[kTopkSortMax];
    const int64_t row = blockIdx.x;
    const uint32_t* sv = sel_vals + row * k;
    const int32_t* si = sel_idx + row * k;
    for (uint32_t i = threadIdx.x; i < npow; i += kTopkSortThreads)
        s[i] = i < k ? ((uint64_t)topk_key(sv[i], largest) << 32) | (uint32_t)~(uint32_t)si[i]
                     : 0ull;
    __syncthreads();
    bitonic_desc(s, npow, kTopkSortThreads);
    for (uint32_t i = threadIdx.x; i < k; i += kTopkSortThreads) {
        const uint64_t c = s[i];
        const uint32_t key = (uint32_t)(c >> 32);
        const uint32_t code = largest ? key : ~key;
        values[row * k + i] = code ^ ((code >> 31) ? 0x80000000u : 0xFFFFFFFFu);
        indices[row * k + i] = (int32_t)~(uint32_t)c;
    }
}

// ---------------------------------------------------------------- gather route

constexpr int64_t kTopkGatherMaxLen = 1 << 17;
constexpr uint32_t kTopkGatherSegs = 16;  // row tiles of the route: 2^17 / 8192 or 16384 / 4096
constexpr uint32_t kTopkCand = 16384;  // candidates sorted in LDS (128 KB)
constexpr int kTopkFinishThreads = 1024;
constexpr uint32_t kTopkSortAll = 2048;  // candidates sorted whole, without the cut to k
constexpr uint32_t kTopkSmallBucket = 128;  // a cut round's bucket finished by one sort
constexpr uint32_t kTopkRankMax = 256;  // kept keys placed by rank instead of sorted
// Outputs per finishing workgroup on the gather route: a row with larger k
// is finished by topk_parts(k) workgroups, each cutting and sorting one
// slice of ranks (smaller sorts, and the chip's other CUs put to work).
constexpr uint32_t kTopkPartKeys = 2048;
__host__ __device__ inline uint32_t topk_parts(uint32_t k) {
    return k > kTopkPartKeys ? (k + kTopkPartKeys - 1) / kTopkPartKeys : 1u;
}
static_assert(kTopkSortMax <= kTopkCand, "the k kept fit the finisher's sort");

// The composite sort key of element i with key `key`: larger keys first,
// equal keys by increasing index.  Every composite is at least 2^31 in its
// low word, so zero pads sort last.
__device__ __forceinline__ uint64_t topk_composite(uint32_t key, uint32_t i) {
    return ((uint64_t)key << 32) | (uint32_t)~i;
}

// Round 0 of the gather route, in two kernels with no per-row arrival (a
// kernel boundary costs less than the arrival atomics): k_topk_count0 stores
// each tile's counts of the top key byte in the tile's own 256 slots, and
// k_topk_bucket, one workgroup per row, adds the row's tile counts per digit
// and leaves in the row's state the digit d whose bucket holds the k-th
// largest key -- fewer than k keys above it, at least k at or above it --
// and k minus the keys above the bucket, and in its gather words the
// candidate count (the keys with a top byte >= d) and a cleared reservation
// counter.  Counting uses one LDS histogram per lane position, shared by the
// waves and padded by a word (copy c, digit d in bank (c + d) mod 32), so the
// lanes of an atomic instruction that hold the same digit -- the top bytes of
// float data take a handful of values -- add to different words.
constexpr int kTopkCopies = 16;
constexpr int kTopkCopyStride = kTopkDigits + 1;
template <class TileT, bool VEC>
__global__ __launch_bounds__(TileT::kThreads) LS_OCCUPANCY4 void k_topk_count0(
    const uint32_t* x, int64_t len, uint32_t segs, bool largest, uint32_t* hist) {
    static_assert(TileT::kThreads >= kTopkDigits, "one thread per digit");
    __shared__ uint32_t s_h[kTopkCopies * kTopkCopyStride];
    for (int i = threadIdx.x; i < kTopkCopies * kTopkCopyStride; i += TileT::kThreads) s_h[i] = 0;
    const int64_t row = blockIdx.x / segs;
    const uint32_t seg = blockIdx.x - (uint32_t)row * segs;
    const int64_t base = (int64_t)seg * TileT::kElems;
    uint32_t v[TileT::J][TileT::V];
    TileT::template load<VEC, true>(x + row * len, len, base, v);
    __syncthreads();  // histograms cleared
    uint32_t* h = s_h + (lane_id() & (kTopkCopies - 1)) * kTopkCopyStride;
    const int32_t valid = (int32_t)(len - base < TileT::kElems ? len - base : TileT::kElems);
#pragma unroll
    for (int j = 0; j < TileT::J; ++j) {
        const int32_t off = (int32_t)TileT::lane_offset(j);
#pragma unroll
        for (int e = 0; e < TileT::V; ++e)
            if (off + e < valid) atomicAdd(&h[topk_key(v[j][e], largest) >> 24], 1u);
    }
    __syncthreads();
    if (threadIdx.x < kTopkDigits) {
        uint32_t t = 0;
#pragma unroll
        for (int q = 0; q < kTopkCopies; ++q) t += s_h[q * kTopkCopyStride + threadIdx.x];
        hist[(int64_t)blockIdx.x * kTopkDigits + threadIdx.x] = t;
    }
}

__global__ __launch_bounds__(kTopkDigits) void k_topk_bucket(const uint32_t* hist, uint32_t segs,
                                                             uint32_t k, uint64_t* state,
                                                             uint64_t* gather, uint32_t* offs,
                                                             uint32_t* rowhist) {
    __shared__ uint32_t s_part[kTopkDigits / kWave];
    __shared__ uint32_t s_d;
    __shared__ uint32_t s_tile[kTopkDigits / kWave][kTopkGatherSegs];
    const int64_t row = blockIdx.x;
    // thread t takes digit 255 - t, so an inclusive scan over t counts the
    // keys with a digit >= its own
    const int t = threadIdx.x;
    const int w = t / kWave;
    const int lane = lane_id();
    const uint32_t* rh = hist + row * segs * kTopkDigits + (kTopkDigits - 1 - t);
    uint32_t c[kTopkGatherSegs];
    uint32_t cnt = 0;
#pragma unroll
    for (uint32_t q = 0; q < kTopkGatherSegs; ++q) {
        c[q] = q < segs ? rh[(int64_t)q * kTopkDigits] : 0u;
        cnt += c[q];
    }
    rowhist[row * kTopkDigits + t] = cnt;  // the row's count of digit 255 - t
    const uint32_t inc = wave_incl_scan(cnt);
    if (lane == kWave - 1) s_part[w] = inc;
    __syncthreads();
    uint32_t before = 0;
    for (int q = 0; q < w; ++q) before += s_part[q];
    const uint32_t at_least = before + inc;  // keys with digit >= 255 - t
    const uint32_t above = at_least - cnt;   // keys with digit > 255 - t
    if (above < k && k <= at_least) {       // exactly one thread (k <= len)
        s_d = (uint32_t)(kTopkDigits - 1 - t);
        state[2 * row] = (uint64_t)(kTopkDigits - 1 - t);
        state[2 * row + 1] = (uint64_t)(k - above);
        gather[2 * row] = at_least;
    }
    __syncthreads();
    // each tile's candidates (its keys with a digit >= d), then their first
    // slots in the row's list: the tiles in order
    const bool keep = (uint32_t)(kTopkDigits - 1 - t) >= s_d;
#pragma unroll
    for (uint32_t q = 0; q < kTopkGatherSegs; ++q) {
        const uint32_t n = wave_sum(keep ? c[q] : 0u);
        if (lane == 0) s_tile[w][q] = n;
    }
    __syncthreads();
    if (t < kWave) {
        uint32_t n = 0;
        if ((uint32_t)lane < segs)
            for (int q = 0; q < kTopkDigits / kWave; ++q) n += s_tile[q][lane];
        const uint32_t incl = wave_incl_scan(n);
        if ((uint32_t)lane < segs) offs[row * kTopkGatherSegs + lane] = incl - n;
    }
}

// Every key of a row whose top digit is at least the bucket's (state after
// round 0), to the row's candidate list (cap slots per row), tile by tile
// from the first slots the bucket kernel left for each tile, in index order
// inside a tile.  Rows with more than cap candidates are left alone.
// Write a tile's candidates -- element (j, e) of this lane when bit j V + e
// of `take` is set, the lane's first at tile slot lpos, total in the tile --
// as keys to ck[0, total) and complemented row indices (base + the element's
// tile offset) to ci[0, total), both clipped to `room` slots.  Up to
// kTopkStage of them are gathered in LDS first (s_ck, s_ci) and written by
// consecutive threads; more go straight from each lane (a uniform choice).
// Every thread of the workgroup calls it.
constexpr uint32_t kTopkStage = 1024;
template <class TileT, class V, class Mask>
__device__ __forceinline__ void stage_candidates(const V& v, Mask take, uint32_t lpos,
                                                 uint32_t total, uint32_t base, uint32_t* ck,
                                                 uint32_t* ci, uint32_t room, uint32_t* s_ck,
                                                 uint32_t* s_ci) {
    const bool staged = total <= kTopkStage;  // uniform
    uint32_t* dk = staged ? s_ck : ck;
    uint32_t* di = staged ? s_ci : ci;
    const uint32_t lim = staged ? kTopkStage : room;
    uint32_t lane0 = base + (uint32_t)TileT::lane_offset(0);
    asm volatile("" : "+v"(lane0));  // no per-chunk offsets kept live from the loads
    if (take) {
#pragma unroll
        for (int j = 0; j < TileT::J; ++j) {
            const uint32_t off = lane0 + (uint32_t)(TileT::lane_offset(j) - TileT::lane_offset(0));
#pragma unroll
            for (int e = 0; e < TileT::V; ++e) {
                if ((take >> (j * TileT::V + e)) & 1u) {
                    if (lpos < lim) {  // lpos < total; checked all the same
                        dk[lpos] = v[j][e];
                        di[lpos] = ~(off + (uint32_t)e);
                    }
                    ++lpos;
                }
            }
        }
    }
    if (!staged) return;
    __syncthreads();
    const uint32_t n = total < room ? total : room;
    for (uint32_t i = threadIdx.x; i < n; i += TileT::kThreads) {
        ck[i] = s_ck[i];
        ci[i] = s_ci[i];
    }
}

template <class TileT, bool VEC>
__global__ __launch_bounds__(TileT::kThreads) LS_OCCUPANCY8 void k_topk_gather(
    const uint32_t* x, int64_t len, uint32_t segs, bool largest, const uint64_t* state,
    const uint64_t* gather, const uint32_t* offs, uint64_t* cand, uint32_t cap) {
    __shared__ uint32_t s_wtot[TileT::WAVES];
    __shared__ uint32_t s_ck[kTopkStage], s_ci[kTopkStage];
    const uint32_t row32 = blockIdx.x / segs;
    const uint32_t seg = blockIdx.x - row32 * segs;
    const int64_t row = row32;
    if ((uint32_t)gather[2 * row] > cap) return;  // uniform: finished the long way
    const uint32_t d = (uint32_t)state[2 * row] & 255u;
    const uint32_t first = offs[row * kTopkGatherSegs + seg];
    const int64_t base = (int64_t)seg * TileT::kElems;
    uint32_t v[TileT::J][TileT::V];
    TileT::template load<VEC, true>(x + row * len, len, base, v);
    const int32_t valid = (int32_t)(len - base < TileT::kElems ? len - base : TileT::kElems);
    static_assert(TileT::J * TileT::V <= 64, "per-lane take masks are 64-bit");
    uint64_t take = 0;
    uint32_t cnt = 0;
#pragma unroll
    for (int j = 0; j < TileT::J; ++j) {
        const int32_t off = (int32_t)TileT::lane_offset(j);
#pragma unroll
        for (int e = 0; e < TileT::V; ++e) {
            const uint32_t key = topk_key(v[j][e], largest);
            const bool t = off + e < valid && (key >> 24) >= d;
            v[j][e] = key;
            take |= (uint64_t)t << (j * TileT::V + e);
            cnt += t ? 1u : 0u;
        }
    }
    // this lane's first slot within the tile: lanes before it in its wave,
    // then the waves before it
    const uint32_t incl = wave_incl_scan(cnt);
    const int w = threadIdx.x / kWave;
    if (lane_id() == kWave - 1) s_wtot[w] = incl;
    __syncthreads();
    uint32_t lpos = incl - cnt, total = 0;  // this lane's first slot in the tile
#pragma unroll
    for (int q = 0; q < TileT::WAVES; ++q) {
        lpos += q < w ? s_wtot[q] : 0u;
        total += s_wtot[q];
    }
    // the row's list: cap keys, then as many complemented indices (the two
    // halves of the composites, in two arrays so that no key needs an aligned
    // register pair of its own)
    uint32_t* ck = reinterpret_cast<uint32_t*>(cand + (int64_t)row * cap);
    uint32_t* ci = ck + cap;
    stage_candidates<TileT>(v, take, lpos, total, (uint32_t)base, ck + first, ci + first,
                            cap - (first < cap ? first : cap), s_ck, s_ci);
}

// The route for small k (rows of up to 2^17 elements, k <= kTopkTileK): one
// read of each row.  Every tile keeps as candidates its keys whose top 16
// bits are at least those of the tile's own k-th largest key.  That is a
// superset of the tile's share of the row's top k: a key below it has k keys
// of its own tile above it.  Two digit rounds over the tile, held in
// registers, find that 16-bit prefix (LDS histograms as in k_topk_count0);
// the tile writes its candidates to its own kTopkTileSlots slots (keys and
// complemented indices, the two halves of their composites) and their number
// to tcount (more than the slots: none written, and the row is finished the
// long way).
constexpr uint32_t kTopkTileK = 256;
constexpr uint32_t kTopkTileSlots = 1024;
static_assert(kTopkTileSlots * kTopkGatherSegs <= kTopkCand, "a row's candidates fit the LDS sort");

// Thread t takes digit 255 - t, the sum of its COPIES histogram copies; an
// inclusive scan over the threads counts the keys with a digit >= its own.
// The thread whose digit's bucket holds the need-th largest counted key (1 <=
// need <= the keys counted) writes the digit and need minus the keys above
// the bucket to *s_out, as digit | rest << 8.
template <int COPIES>
__device__ __forceinline__ void tile_bucket(const uint32_t* s_h, uint32_t need, uint32_t* s_part,
                                            uint32_t* s_out) {
    const int t = threadIdx.x;
    const int w = t / kWave;
    uint32_t c = 0;
    if (t < kTopkDigits) {
#pragma unroll
        for (int q = 0; q < COPIES; ++q) c += s_h[q * kTopkCopyStride + (kTopkDigits - 1 - t)];
    }
    const uint32_t inc = wave_incl_scan(c);
    if (t < kTopkDigits && lane_id() == kWave - 1) s_part[w] = inc;
    __syncthreads();
    if (t < kTopkDigits) {
        uint32_t before = 0;
        for (int q = 0; q < w; ++q) before += s_part[q];
        const uint32_t at_least = before + inc, above = at_least - c;
        if (above < need && need <= at_least)
            *s_out = (uint32_t)(kTopkDigits - 1 - t) | ((need - above) << 8);
    }
}

template <class TileT, bool VEC>
__global__ __launch_bounds__(TileT::kThreads) LS_OCCUPANCY8 void k_topk_tilesel(
    const uint32_t* x, int64_t len, uint32_t segs, uint32_t k, bool largest, uint64_t* cand,
    uint32_t* tcount) {
    static_assert(TileT::kThreads >= kTopkDigits, "one thread per digit");
    // round 1 counts only the keys of one round-0 bucket: fewer copies, so
    // that the LDS of 8 workgroups fits a CU (with at most 64 VGPRs, 8 waves
    // per SIMD: every tile of a 128 x 131072 call resident at once)
    constexpr int kCopies1 = 2;
    constexpr int kHist = kTopkCopies * kTopkCopyStride, kHist1 = kCopies1 * kTopkCopyStride;
    __shared__ uint32_t s_h[kHist];
    __shared__ uint32_t s_h1[kHist1];
    __shared__ uint32_t s_part[kTopkDigits / kWave];
    __shared__ uint32_t s_wtot[TileT::WAVES];
    __shared__ uint32_t s_sel;
    for (int i = threadIdx.x; i < kHist; i += TileT::kThreads) s_h[i] = 0;
    for (int i = threadIdx.x; i < kHist1; i += TileT::kThreads) s_h1[i] = 0;
    const int64_t row = blockIdx.x / segs;
    const uint32_t seg = blockIdx.x - (uint32_t)row * segs;
    const int64_t base = (int64_t)seg * TileT::kElems;
    uint32_t v[TileT::J][TileT::V];
    TileT::template load<VEC, true>(x + row * len, len, base, v);
    const int32_t valid = (int32_t)(len - base < TileT::kElems ? len - base : TileT::kElems);
    __syncthreads();  // histograms cleared
    uint32_t* h = s_h + (lane_id() & (kTopkCopies - 1)) * kTopkCopyStride;
    // bit j V + e: element (j, e) of this lane lies in the row (one register;
    // opaque, so that the compiler keeps no per-element flags beside it)
    using Mask = typename std::conditional<(TileT::J * TileT::V > 32), uint64_t, uint32_t>::type;
    static_assert(TileT::J * TileT::V <= 64, "per-lane masks of at most 64 bits");
    Mask inrow = 0;
#pragma unroll
    for (int j = 0; j < TileT::J; ++j) {
        const int32_t off = (int32_t)TileT::lane_offset(j);
#pragma unroll
        for (int e = 0; e < TileT::V; ++e)
            inrow |= (Mask)(off + e < valid ? 1u : 0u) << (j * TileT::V + e);
    }
    asm volatile("" : "+v"(inrow));
    // round 0: the top byte of every key of the tile.  Positions past the
    // row's end count as key 0, the smallest: need <= valid, so they do not
    // move the need-th largest key, and the candidates are taken below with
    // the bound checked.
#pragma unroll
    for (int j = 0; j < TileT::J; ++j) {
#pragma unroll
        for (int e = 0; e < TileT::V; ++e) {
            const uint32_t key = topk_key(v[j][e], largest);
            v[j][e] = (inrow >> (j * TileT::V + e)) & 1u ? key : 0u;
            asm volatile("" : "+v"(v[j][e]));  // the unmasked key is dead here
            atomicAdd(&h[v[j][e] >> 24], 1u);
        }
    }
    __syncthreads();
    const uint32_t need = k < (uint32_t)valid ? k : (uint32_t)valid;
    tile_bucket<kTopkCopies>(s_h, need, s_part, &s_sel);
    __syncthreads();  // s_sel written
    const uint32_t d = s_sel & 255u, need1 = s_sel >> 8;
    // round 1: the second byte of the keys in bucket d
    uint32_t* h1 = s_h1 + (lane_id() & (kCopies1 - 1)) * kTopkCopyStride;
#pragma unroll
    for (int j = 0; j < TileT::J; ++j) {
#pragma unroll
        for (int e = 0; e < TileT::V; ++e)
            if ((v[j][e] >> 24) == d) atomicAdd(&h1[(v[j][e] >> 16) & 255u], 1u);
    }
    __syncthreads();
    tile_bucket<kCopies1>(s_h1, need1, s_part, &s_sel);
    __syncthreads();
    const uint32_t p16 = (d << 8) | (s_sel & 255u);
    Mask take = 0;
    uint32_t cnt = 0;
#pragma unroll
    for (int j = 0; j < TileT::J; ++j) {
#pragma unroll
        for (int e = 0; e < TileT::V; ++e) {
            const bool t = ((inrow >> (j * TileT::V + e)) & 1u) && (v[j][e] >> 16) >= p16;
            take |= (Mask)(t ? 1u : 0u) << (j * TileT::V + e);
            cnt += t ? 1u : 0u;
        }
    }
    // this lane's first slot within the tile: lanes before it in its wave,
    // then the waves before it
    const uint32_t incl = wave_incl_scan(cnt);
    const int w = threadIdx.x / kWave;
    if (lane_id() == kWave - 1) s_wtot[w] = incl;
    __syncthreads();
    uint32_t lpos = incl - cnt, total = 0;  // this lane's first slot in the tile
#pragma unroll
    for (int q = 0; q < TileT::WAVES; ++q) {
        lpos += q < w ? s_wtot[q] : 0u;
        total += s_wtot[q];
    }
    if (threadIdx.x == 0) tcount[blockIdx.x] = total;
    if (total > kTopkTileSlots) return;  // uniform: the row goes the long way
    // The tile's slots: kTopkTileSlots keys, then as many complemented
    // indices (two arrays rather than 64-bit composites, so that no key needs
    // an aligned register pair of its own); staged in the round-0 histogram's
    // LDS, which is free by now.
    static_assert(kTopkTileSlots <= kTopkStage && 2 * kTopkStage <= kHist, "staging room");
    uint32_t* ck = reinterpret_cast<uint32_t*>(cand + (int64_t)blockIdx.x * kTopkTileSlots);
    stage_candidates<TileT>(v, take, lpos, total, (uint32_t)base, ck, ck + kTopkTileSlots,
                            kTopkTileSlots, s_h, s_h + kTopkStage);
}

// The same network on npow keys held in registers, E per thread (thread t:
// positions t E .. t E + E - 1; positions at or past npow are padding that
// never meets a real key): strides below E inside the thread, strides below
// 64 E between the lanes of a wavefront (shuffles, no barrier), larger
// strides through LDS (s, at least max(npow, E * nthreads) slots).
//
// `run` (a power of two, at most npow): sort each block of `run` positions,
// every block descending (run = npow: the whole array).
template <int E>
__device__ __forceinline__ void bitonic_desc_regs(uint64_t (&v)[E], uint64_t* s, uint32_t npow,
                                                  uint32_t nthreads, uint32_t run) {
    const uint32_t t = threadIdx.x;
    for (uint32_t size = 2; size <= run; size <<= 1) {
        // blocks of `size` alternate direction, except in the last merge
        const bool all_desc = size == run;
        uint32_t stride = size >> 1;
        if (stride >= (uint32_t)(kWave * E)) {  // uniform
#pragma unroll
            for (int e = 0; e < E; ++e) s[t * E + e] = v[e];
            __syncthreads();
            for (; stride >= (uint32_t)(kWave * E); stride >>= 1) {
                for (uint32_t q = t; q < npow / 2; q += nthreads) {
                    const uint32_t i = 2 * q - (q & (stride - 1));
                    const uint32_t j = i + stride;
                    const uint64_t a = s[i], b = s[j];
                    const uint64_t hi = a > b ? a : b, lo = a > b ? b : a;
                    const bool desc = all_desc || (i & size) == 0;
                    s[i] = desc ? hi : lo;
                    s[j] = desc ? lo : hi;
                }
                __syncthreads();
            }
#pragma unroll
            for (int e = 0; e < E; ++e) v[e] = s[t * E + e];  // this thread's own slots
        }
        for (; stride >= (uint32_t)E; stride >>= 1) {
            const int lanes = (int)(stride / E);
            // stride >= E: the thread's positions share their stride and size
            // bits, so one choice per stage: keep the larger of each pair at
            // the lower position of a descending block, the smaller otherwise
            const uint32_t p0 = t * E;
            const bool keep_max = ((p0 & stride) == 0) == (all_desc || (p0 & size) == 0);
#pragma unroll
            for (int e = 0; e < E; ++e) {
                const uint64_t w = __shfl_xor(v[e], lanes);
                v[e] = ((v[e] > w) != keep_max) ? w : v[e];
            }
        }
        // strides below E (those below size), inside the thread
#pragma unroll
        for (int st = E / 2; st >= 1; st /= 2) {
            if ((uint32_t)st < size) {  // uniform
#pragma unroll
                for (int e = 0; e < E; ++e) {
                    if ((e & st) == 0) {
                        const int e2 = e | st;
                        const bool desc = all_desc || ((t * E + e) & size) == 0;
                        const uint64_t a = v[e], b = v[e2];
                        const bool sw = (a < b) == desc;
                        v[e] = sw ? b : a;
                        v[e2] = sw ? a : b;
                    }
                }
            }
        }
    }
}

// Merge path: with runs of L descending keys in src, thread t's E outputs
// of the merged runs of 2 L (positions t E .. t E + E - 1): the number of
// them taken from the first run by a binary search, then E merge steps.
// Keys are distinct (composites), so there are no ties.
template <int E>
__device__ __forceinline__ void merge_desc(const uint64_t* src, uint32_t L, uint64_t (&out)[E]) {
    const uint32_t i0 = threadIdx.x * E;
    const uint32_t pair = i0 / (2 * L);
    const uint32_t r = i0 - pair * 2 * L;
    const uint64_t* A = src + pair * 2 * L;
    const uint64_t* B = A + L;
    uint32_t lo = r > L ? r - L : 0, hi = r < L ? r : L;
    while (lo < hi) {  // A's share of the r largest
        const uint32_t mid = (lo + hi) / 2;
        if (A[mid] > B[r - mid - 1]) lo = mid + 1; else hi = mid;
    }
    uint32_t a = lo, b = r - lo;
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const bool take_a = b >= L || (a < L && A[a] > B[b]);
        out[e] = take_a ? A[a] : B[b];
        a += take_a ? 1u : 0u;
        b += take_a ? 0u : 1u;
    }
}

// For i < n (1 <= n <= kTopkRankMax, a holding at least n rounded up to a
// power of two >= 64 slots, distinct keys): s_rank[i] = the number of keys
// of a[0, n) above a[i], its place in descending order.  Each of the
// workgroup's kTopkFinishThreads threads counts over one of kT / P slices
// for one key (P: n rounded up to a power of two, at least 64), so that all
// waves share the work and the slice loads of a wave are one address.  Ends
// with a barrier.
template <uint32_t P>
__device__ __forceinline__ void rank_keys_p(const uint64_t* a, uint32_t n, uint32_t* s_rank) {
    constexpr uint32_t kT = kTopkFinishThreads;
    constexpr uint32_t L = P * P / kT;  // 64: 4, 128: 16, 256: 64
    static_assert(P <= kT && L >= 1, "every key with a thread");
    const uint32_t i = threadIdx.x % P, q = threadIdx.x / P;
    if (threadIdx.x < P) s_rank[threadIdx.x] = 0;
    const uint64_t me = a[i];
    __syncthreads();  // s_rank cleared
    uint32_t above = 0;
    const uint32_t j0 = q * L;
    if (j0 < n) {  // uniform in the wave
#pragma unroll
        for (uint32_t u = 0; u < L; ++u) {
            const uint32_t j = j0 + u;  // < P
            const uint64_t o = a[j];
            above += (j < n && o > me) ? 1u : 0u;
        }
    }
    if (i < n && above) atomicAdd(&s_rank[i], above);
    __syncthreads();
}
__device__ __forceinline__ void rank_keys(const uint64_t* a, uint32_t n, uint32_t* s_rank) {
    static_assert(kTopkRankMax == 256, "the sizes below");
    if (n <= 64)
        rank_keys_p<64>(a, n, s_rank);
    else if (n <= 128)
        rank_keys_p<128>(a, n, s_rank);
    else
        rank_keys_p<256>(a, n, s_rank);
}

// One workgroup per row: the k largest keys of the row, in order.  A row
// whose candidates were gathered sorts them and keeps the first k.  Any
// other row is finished here: three more digit rounds inside the bucket
// (histograms in LDS, over the row) give the k-th key T and kk, the number
// of keys equal to T in the top k; a walk over the row in index order takes
// every key above T and the first kk equal to T; those k are sorted.
// CAP slots of LDS (a power of two, at least cap) hold the keys to sort.
//
// TILES (the small-k route): the candidates are the row's tiles' lists
// (tcount: each tile's count, cand: kTopkTileSlots slots per tile, as
// k_topk_tilesel lays them out), and no digit of the k-th key is known yet,
// so the rounds start from the top byte.
template <uint32_t CAP, bool TILES>
__global__ __launch_bounds__(kTopkFinishThreads) void k_topk_finish(
    const uint32_t* x, int64_t len, uint32_t k, bool largest, const uint64_t* state,
    const uint64_t* gather, const uint64_t* cand, uint32_t cap, uint32_t segs,
    const uint32_t* tcount, const uint32_t* rowhist, uint32_t* values, int32_t* indices) {
    static_assert(CAP <= kTopkCand && (CAP & (CAP - 1)) == 0, "LDS sort size");
    __shared__ uint64_t s[CAP];
    // digit counts: one copy per lane position, as in k_topk_count0 (the
    // keys of a round share few digits)
    __shared__ uint32_t s_h[kTopkCopies * kTopkCopyStride];
    __shared__ uint32_t s_part[kTopkFinishThreads / kWave];
    __shared__ uint32_t s_prefix, s_kk, s_n, s_qbase, s_bucket, s_nsmall, s_m, s_over;
    __shared__ uint64_t s_prefix64;
    __shared__ uint32_t s_dig[2], s_dkk[2];
    __shared__ uint64_t s_small[kTopkSmallBucket];
    __shared__ uint32_t s_off[kTopkGatherSegs], s_cnt[kTopkGatherSegs];
    __shared__ uint32_t s_rank[kTopkRankMax];
    constexpr uint32_t kT = kTopkFinishThreads;
    static_assert(!TILES || kTopkTileSlots <= kT, "one tile slot per thread");
    // A row's outputs are split between topk_parts(k) workgroups: part q
    // writes ranks [lo, hi) = [q P, min((q + 1) P, k)), P = kTopkPartKeys.
    const uint32_t parts = TILES ? 1u : topk_parts(k);
    const int64_t row = blockIdx.x / parts;
    const uint32_t part = blockIdx.x - (uint32_t)row * parts;
    uint32_t lo = part * kTopkPartKeys;
    uint32_t hi = k - lo < kTopkPartKeys ? k : lo + kTopkPartKeys;
    // the row's top-byte counts (thread t: digit 255 - t), loaded under the
    // candidate loads: they place a slice's boundaries without a digit round
    // over the candidates (the keys with the top byte of the k-th or more are
    // all candidates, and every boundary rank is at most k)
    uint32_t rh = 0;
    if (!TILES && parts > 1 && threadIdx.x < kTopkDigits)
        rh = rowhist[row * kTopkDigits + threadIdx.x];
    const int w = threadIdx.x / kWave;
    const int lane = lane_id();
    uint32_t* hcopy = s_h + (lane & (kTopkCopies - 1)) * kTopkCopyStride;
    auto digit_count = [&](int t) {  // thread t: digit 255 - t, all copies
        uint32_t c = 0;
        if (t < kTopkDigits) {
#pragma unroll
            for (int q = 0; q < kTopkCopies; ++q) c += s_h[q * kTopkCopyStride + (kTopkDigits - 1 - t)];
        }
        return c;
    };
    uint32_t m;
    bool fits;
    if constexpr (TILES) {
        // the row's candidates: each tile's count and first slot in LDS
        if (threadIdx.x < kWave) {
            const uint32_t c = (uint32_t)lane < segs ? tcount[row * segs + lane] : 0u;
            const uint64_t over = __ballot(c > kTopkTileSlots);
            const uint32_t incl = wave_incl_scan(c);
            if ((uint32_t)lane < kTopkGatherSegs) {
                s_off[lane] = incl - c;
                s_cnt[lane] = c;
            }
            if (lane == kWave - 1) {
                s_m = incl;
                s_over = over != 0 ? 1u : 0u;
            }
        }
        __syncthreads();
        m = s_m;
        fits = s_over == 0;
    } else {
        m = (uint32_t)gather[2 * row];
        fits = m <= cap;
        if (!fits) {  // uniform: part 0 finishes the row the long way, all k ranks
            if (part != 0) return;
            hi = k;
        }
    }
    const uint32_t sort_all = TILES ? kTopkRankMax : kTopkSortAll;
    if (fits) {
        // The k largest of the m candidates.  Up to kTopkSortAll of them are
        // all sorted (the first k are the answer); more are first cut to k:
        // the k-th largest composite C by seven more digit rounds over the
        // candidates in LDS (the first digit, the key's top byte, is the
        // bucket's), then the composites >= C (exactly k: composites are
        // distinct) to the front.
        // every candidate load in flight at once, then to LDS for the rounds
        // Slot e of this thread: candidate t + e kT of the row's list, or
        // (TILES) candidate t of tile e, which goes to LDS slot off_e + t.
        constexpr int kPer = CAP / kTopkFinishThreads > 0 ? CAP / kTopkFinishThreads : 1;
        auto slot_valid = [&](int e) {
            if constexpr (TILES)
                return (uint32_t)e < segs && threadIdx.x < s_cnt[e];
            else
                return threadIdx.x + e * kT < m;
        };
        auto slot_lds = [&](int e) {
            if constexpr (TILES)
                return s_off[e] + threadIdx.x;
            else
                return threadIdx.x + e * kT;
        };
        uint64_t mine[kPer];
        uint32_t vmask = 0;  // bit e: slot e holds a candidate
#pragma unroll
        for (int e = 0; e < kPer; ++e) {
            mine[e] = 0ull;
            if (slot_valid(e)) {
                vmask |= 1u << e;
                if constexpr (TILES) {
                    // tile e's slot t: its key and complemented index
                    const uint32_t* ck = reinterpret_cast<const uint32_t*>(
                        cand + ((int64_t)row * segs + e) * kTopkTileSlots);
                    mine[e] = ((uint64_t)ck[threadIdx.x] << 32) | ck[kTopkTileSlots + threadIdx.x];
                } else {
                    // the row's list: cap keys, then the complemented indices
                    const uint32_t* ck = reinterpret_cast<const uint32_t*>(cand + row * cap);
                    const uint32_t i = threadIdx.x + e * kT;
                    mine[e] = ((uint64_t)ck[i] << 32) | ck[cap + i];
                }
            }
        }
#pragma unroll
        for (int e = 0; e < kPer; ++e)
            if ((vmask >> e) & 1u) s[slot_lds(e)] = mine[e];
        // The kk-th largest of the candidates whose top 8 r0 bits are
        // `prefix`: digit rounds from digit r0 on, each keeping the bucket
        // that holds it, until the last digit or a bucket small enough to
        // rank.
        auto find_kth = [&](uint32_t kk, int r0, uint64_t prefix) -> uint64_t {
            for (int r = r0; r < 8; ++r) {
                for (uint32_t i = threadIdx.x; i < kTopkCopies * kTopkCopyStride; i += kT)
                    s_h[i] = 0;
                __syncthreads();  // also: the candidates are in LDS
                const int hs = 64 - 8 * r, ds = 56 - 8 * r;
                for (uint32_t i = threadIdx.x; i < m; i += kT) {
                    const uint64_t c = s[i];
                    if (r == 0 || (c >> hs) == prefix)
                        atomicAdd(&hcopy[(uint32_t)(c >> ds) & 255u], 1u);
                }
                __syncthreads();
                const int t = threadIdx.x;
                const uint32_t c = digit_count(t);
                const uint32_t inc = wave_incl_scan(c);
                if (t < kTopkDigits && lane == kWave - 1) s_part[w] = inc;
                __syncthreads();
                if (t < kTopkDigits) {
                    uint32_t before = 0;
                    for (int q = 0; q < w; ++q) before += s_part[q];
                    const uint32_t at_least = before + inc, above = at_least - c;
                    if (above < kk && kk <= at_least) {  // exactly one thread
                        s_prefix64 = (prefix << 8) | (uint32_t)(kTopkDigits - 1 - t);
                        s_kk = kk - above;
                        s_bucket = c;
                    }
                }
                __syncthreads();
                prefix = s_prefix64;
                kk = s_kk;
                if (s_bucket <= kTopkSmallBucket) {  // uniform
                    // A bucket this small is finished in one step instead of
                    // more rounds: its composites are gathered and ranked, and
                    // the one with kk - 1 above it is the k-th largest composite
                    // of the row.
                    const int hs2 = 56 - 8 * r;  // the new prefix's shift
                    const uint32_t nb = s_bucket;  // >= kk >= 1
                    if (threadIdx.x == 0) s_nsmall = 0;
                    __syncthreads();
                    for (uint32_t i = threadIdx.x; i < m; i += kT) {
                        const uint64_t c2 = s[i];
                        if ((c2 >> hs2) == prefix) {
                            const uint32_t pos = atomicAdd(&s_nsmall, 1u);
                            if (pos < kTopkSmallBucket) s_small[pos] = c2;  // below the bucket size
                        }
                    }
                    __syncthreads();
                    rank_keys(s_small, nb, s_rank);
                    if (threadIdx.x < nb && s_rank[threadIdx.x] == kk - 1)  // exactly one
                        s_prefix64 = s_small[threadIdx.x];
                    __syncthreads();
                    prefix = s_prefix64;
                    break;
                }
            }
            return prefix;
        };
        const bool cut = parts > 1 || (m > k && m > sort_all);  // uniform
        // Cut: the composites of ranks [lo, hi), those in [C_hi, C_lo) with
        // C_r the r-th largest (C_0 above every key).  C_k from the bucket
        // the count round chose (TILES: from the top byte on), other ranks
        // from the top byte on.
        uint64_t c_hi = 0, c_lo = ~0ull;
        if (cut && parts > 1) {
            // the top bytes of C_hi and C_lo and their ranks within those
            // bytes' buckets, from the row's counts
            const int t = threadIdx.x;
            const uint32_t c = t < kTopkDigits ? rh : 0u;
            const uint32_t inc = wave_incl_scan(c);
            if (t < kTopkDigits && lane == kWave - 1) s_part[w] = inc;
            __syncthreads();
            if (t < kTopkDigits) {
                uint32_t before = 0;
                for (int q = 0; q < w; ++q) before += s_part[q];
                const uint32_t at_least = before + inc, above = at_least - c;
                const uint32_t tgt[2] = {hi, lo};
#pragma unroll
                for (int q = 0; q < 2; ++q) {
                    if (above < tgt[q] && tgt[q] <= at_least) {  // one thread each (lo: if > 0)
                        s_dig[q] = (uint32_t)(kTopkDigits - 1 - t);
                        s_dkk[q] = tgt[q] - above;
                    }
                }
            }
            __syncthreads();
            const uint32_t d_hi = s_dig[0], kk_hi = s_dkk[0], d_lo = s_dig[1], kk_lo = s_dkk[1];
            c_hi = find_kth(kk_hi, 1, d_hi);
            if (part != 0) c_lo = find_kth(kk_lo, 1, d_lo);
        } else if (cut) {
            c_hi = TILES ? find_kth(k, 0, 0ull)
                         : find_kth((uint32_t)state[2 * row + 1], 1,
                                    (uint32_t)state[2 * row] & 255u);
        }
        // Each thread still holds its candidates in `mine`.  Cut: the kept
        // ones go to s[0, hi - lo), each thread's after those of the threads
        // before it (a workgroup scan).  Otherwise all m are in s[0, m)
        // already.
        if (cut) {
            uint32_t keep = 0, cnt = 0;
#pragma unroll
            for (int e = 0; e < kPer; ++e) {
                const bool kp = ((vmask >> e) & 1u) && mine[e] >= c_hi && mine[e] < c_lo;
                keep |= (kp ? 1u : 0u) << e;
                cnt += kp ? 1u : 0u;
            }
            const uint32_t inc = wave_incl_scan(cnt);
            if (lane == kWave - 1) s_part[w] = inc;
            __syncthreads();  // also: every round's reads of s are done
            uint32_t pos = inc - cnt;
#pragma unroll
            for (int q = 0; q < (int)(kT / kWave); ++q) pos += q < w ? s_part[q] : 0u;
#pragma unroll
            for (int e = 0; e < kPer; ++e) {
                if ((keep >> e) & 1u) {
                    if (pos < cap) s[pos] = mine[e];  // pos < hi - lo; checked all the same
                    ++pos;
                }
            }
        }
    } else {
        const uint32_t* xr = x + row * len;
        uint32_t prefix = TILES ? 0u : (uint32_t)state[2 * row];
        uint32_t kk = TILES ? k : (uint32_t)state[2 * row + 1];
        for (int r = TILES ? 0 : 1; r < 4; ++r) {
            for (uint32_t i = threadIdx.x; i < kTopkCopies * kTopkCopyStride; i += kT) s_h[i] = 0;
            __syncthreads();
            const int hs = 32 - 8 * r, ds = 24 - 8 * r;
            for (int64_t i = threadIdx.x; i < len; i += kT) {
                const uint32_t key = topk_key(xr[i], largest);
                if (r == 0 || (key >> hs) == prefix) atomicAdd(&hcopy[(key >> ds) & 255u], 1u);
            }
            __syncthreads();
            // thread t takes digit 255 - t: an inclusive scan over t counts the
            // keys with a digit >= its own
            const int t = threadIdx.x;
            const uint32_t c = digit_count(t);
            const uint32_t inc = wave_incl_scan(c);
            if (t < kTopkDigits && lane == kWave - 1) s_part[w] = inc;
            __syncthreads();
            if (t < kTopkDigits) {
                uint32_t before = 0;
                for (int q = 0; q < w; ++q) before += s_part[q];
                const uint32_t at_least = before + inc, above = at_least - c;
                if (above < kk && kk <= at_least) {  // exactly one thread
                    s_prefix = (prefix << 8) | (uint32_t)(kTopkDigits - 1 - t);
                    s_kk = kk - above;
                }
            }
            __syncthreads();
            prefix = s_prefix;
            kk = s_kk;
            __syncthreads();  // s_prefix / s_kk rewritten by the next round
        }
        // prefix is now the k-th key T: take every key above it and the
        // first kk equal to it, in index order
        if (threadIdx.x == 0) s_n = s_qbase = 0;
        __syncthreads();
        for (int64_t c0 = 0; c0 < len; c0 += kT) {
            const int64_t i = c0 + threadIdx.x;
            const uint32_t key = i < len ? topk_key(xr[i], largest) : 0u;
            const bool a = i < len && key > prefix, q = i < len && key == prefix;
            const uint64_t qb = __ballot(q);
            if (lane == 0) s_part[w] = (uint32_t)__builtin_popcountll(qb);
            __syncthreads();
            uint32_t r = s_qbase + __builtin_amdgcn_mbcnt_hi((uint32_t)(qb >> 32),
                                                             __builtin_amdgcn_mbcnt_lo((uint32_t)qb, 0));
            uint32_t chunk = 0;
            for (int q2 = 0; q2 < (int)(kT / kWave); ++q2) {
                if (q2 < w) r += s_part[q2];
                chunk += s_part[q2];
            }
            if (a || (q && r < kk)) {
                const uint32_t pos = atomicAdd(&s_n, 1u);  // below k; checked all the same
                if (pos < cap) s[pos] = topk_composite(key, (uint32_t)i);
            }
            __syncthreads();
            if (threadIdx.x == 0) s_qbase += chunk;
            __syncthreads();
        }
    }
    // the n kept keys are s[0, n): this part's hi - lo (all of them, n >= k,
    // when the candidates were sorted whole); outputs from rank lo on
    const uint32_t n = (fits && m <= sort_all) ? m : hi - lo;
    auto emit = [&](uint32_t p0, uint64_t c) {  // output lo + p0 (< k): composite c
        const uint32_t p = lo + p0;
        const uint32_t key = (uint32_t)(c >> 32);
        const uint32_t code = largest ? key : ~key;
        values[row * k + p] = code ^ ((code >> 31) ? 0x80000000u : 0xFFFFFFFFu);
        indices[row * k + p] = (int32_t)~(uint32_t)c;
    };
    __syncthreads();
    if (n <= kTopkRankMax) {  // uniform
        // Few keys: each goes straight to its rank, the number of kept keys
        // above it (the composites are distinct).
        rank_keys(s, n, s_rank);
        if (threadIdx.x < n) {
            const uint32_t r = s_rank[threadIdx.x];
            if (r < hi - lo) emit(r, s[threadIdx.x]);
        }
        return;
    }
    if constexpr (TILES) return;  // n <= k <= kTopkRankMax
    // more: sorted in registers, E per thread
    uint32_t npow = 1;
    while (npow < n) npow <<= 1;
    auto sort_out = [&](auto e_c) {
        constexpr int E = decltype(e_c)::value;
        static_assert((uint32_t)E * kT <= CAP || E == 1, "LDS slots for the register sort");
        uint64_t v[E];
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const uint32_t p = threadIdx.x * E + e;
            v[e] = p < n ? s[p] : 0ull;
        }
        __syncthreads();  // every kept key read before the sort writes LDS
        const uint32_t wrun = (uint32_t)(kWave * E);
        if (npow > wrun) {
            // each wavefront's run of 64 E keys sorted in registers, then
            // merge levels through LDS (threads past npow merge padding
            // inside s[0, max(npow, E * kT)) and are never read)
            bitonic_desc_regs<E>(v, s, npow, kT, wrun);
            for (uint32_t L = wrun; L < npow; L <<= 1) {
#pragma unroll
                for (int e = 0; e < E; ++e) s[threadIdx.x * E + e] = v[e];
                __syncthreads();
                merge_desc<E>(s, L, v);
                __syncthreads();  // s is rewritten by the next level
            }
        } else {
            bitonic_desc_regs<E>(v, s, npow, kT, npow);
        }
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const uint32_t p = threadIdx.x * E + e;
            if (p < hi - lo) emit(p, v[e]);
        }
    };
    if (npow <= kT)
        sort_out(std::integral_constant<int, 1>{});
    else if (npow <= 2 * kT)
        sort_out(std::integral_constant<int, 2>{});
    else if (CAP >= 4 * kT && npow <= 4 * kT)
        sort_out(std::integral_constant<int, (CAP >= 4 * kT ? 4 : 1)>{});
    else
        sort_out(std::integral_constant<int, (CAP >= 8 * kT ? 8 : 1)>{});
}

// ---------------------------------------------------------------- launch

// Workspace: header | two look-back chains (rows x segments words each) |
// digit counts (rows x segments x 256) | row states (2 words) | arrival
// counters; the final radix sort (k > kTopkSortMax) reuses the front.
// Scratch: the k kept values and indices per row, and for the radix sort its
// two ping-pong buffers.
static size_t align256(size_t b) { return (b + 255) / 256 * 256; }
// The gather route: rows of at most kTopkGatherMaxLen with k <= kTopkSortMax,
// its count round on tiles of at most 8192 (more workgroups for the one read
// from HBM).
static bool topk_gather_route(int64_t len, int64_t k) {
    return len <= kTopkGatherMaxLen && k <= kTopkSortMax;
}
static int64_t topk_gather_tile(int64_t len) { return len > 16384 ? 8192 : 4096; }
// The small-k route (one read of each row): the gather route's rows and tiles.
static bool topk_tiles_route(int64_t len, int64_t k) {
    return topk_gather_route(len, k) && k <= kTopkTileK;
}
static uint32_t topk_tiles_segs(int64_t len) {
    return (uint32_t)((len + topk_gather_tile(len) - 1) / topk_gather_tile(len));
}
static uint32_t topk_cap(int64_t len) {
    return (uint32_t)(len < (int64_t)kTopkCand ? len : (int64_t)kTopkCand);
}
struct TopkLayout {
    size_t hist, state, arrivals, gather, offs, rowhist, end;
};
static TopkLayout topk_layout(int64_t rows, int64_t len, int64_t k) {
    const int64_t t = topk_gather_route(len, k) ? topk_gather_tile(len) : row_tile(len);
    const size_t tiles = (size_t)rows * (size_t)((len + t - 1) / t);
    TopkLayout l;
    l.hist = align256(kWsHeader + 2 * tiles * sizeof(uint64_t));
    l.state = align256(l.hist + tiles * kTopkDigits * sizeof(uint32_t));
    l.arrivals = l.state + (size_t)rows * 2 * sizeof(uint64_t);
    l.gather = l.arrivals + (size_t)rows * sizeof(uint64_t);
    l.offs = l.gather + (size_t)rows * 2 * sizeof(uint64_t);
    const bool g = topk_gather_route(len, k);
    l.rowhist = l.offs + (g ? (size_t)rows * kTopkGatherSegs * 4 : 0);
    l.end = l.rowhist + (g ? (size_t)rows * kTopkDigits * 4 : 0);
    return l;
}
size_t topk_ws_bytes(int64_t rows, int64_t len, int64_t k) {
    const size_t a = topk_layout(rows, len, k).end;
    const size_t b = k > kTopkSortMax ? radix_rows_ws_bytes(rows, k) : 0;
    return a > b ? a : b;
}
size_t topk_scratch_bytes(int64_t rows, int64_t len, int64_t k) {
    if (topk_tiles_route(len, k))
        return align256((size_t)rows * topk_tiles_segs(len) * kTopkTileSlots * sizeof(uint64_t));
    if (topk_gather_route(len, k)) return align256((size_t)rows * topk_cap(len) * sizeof(uint64_t));
    return (k > kTopkSortMax ? 4 : 2) * align256((size_t)rows * (size_t)k * 4);
}

template <class G>
static hipError_t topk_select(bool vec, const uint32_t* x, int64_t rows, int64_t len, int64_t k,
                              bool largest, uint32_t* sel_vals, int32_t* sel_idx, void* ws,
                              hipStream_t stream) {
    using TV = RowTile<uint32_t, G, true>;
    using TU = RowTile<uint32_t, G, false>;
    static_assert(TV::kElems == TU::kElems, "one tile size per geometry");
    const uint32_t segs = (uint32_t)((len + TV::kElems - 1) / TV::kElems);
    const uint32_t nt = (uint32_t)(rows * segs);
    const unsigned threads = vec ? TV::kThreads : TU::kThreads;
    char* w = reinterpret_cast<char*>(ws);
    const TopkLayout l = topk_layout(rows, len, k);
    uint32_t* hist = reinterpret_cast<uint32_t*>(w + l.hist);
    uint64_t* state = reinterpret_cast<uint64_t*>(w + l.state);
    uint64_t* arrivals = reinterpret_cast<uint64_t*>(w + l.arrivals);
    const uint32_t kk = (uint32_t)k;
    hipLaunchKernelGGL((vec ? k_topk_hist<TV, true, 0> : k_topk_hist<TU, false, 0>), dim3(nt),
                       dim3(threads), 0, stream, x, len, segs, kk, largest, hist, state, arrivals);
    hipLaunchKernelGGL((vec ? k_topk_hist<TV, true, 1> : k_topk_hist<TU, false, 1>), dim3(nt),
                       dim3(threads), 0, stream, x, len, segs, kk, largest, hist, state, arrivals);
    hipLaunchKernelGGL((vec ? k_topk_hist<TV, true, 2> : k_topk_hist<TU, false, 2>), dim3(nt),
                       dim3(threads), 0, stream, x, len, segs, kk, largest, hist, state, arrivals);
    hipLaunchKernelGGL((vec ? k_topk_hist<TV, true, 3> : k_topk_hist<TU, false, 3>), dim3(nt),
                       dim3(threads), 0, stream, x, len, segs, kk, largest, hist, state, arrivals);
    // The split keeps its flags and the tile's packed counts in registers as
    // well: it takes the tile shape with half the chunks and twice the waves
    // (16-byte loads still when aligned).
    uint64_t* status = reinterpret_cast<uint64_t*>(w + kWsHeader);
    hipLaunchKernelGGL((vec ? k_topk_select<TU, true> : k_topk_select<TU, false>), dim3(nt),
                       dim3(TU::kThreads), 0, stream, x, len, segs, nt, kk, largest,
                       (const uint64_t*)state, sel_vals, sel_idx, reinterpret_cast<WsHeader*>(ws),
                       status, (int64_t)2 * nt);
    return hipGetLastError();
}

template <class G>
static hipError_t topk_gather(bool vec, const uint32_t* x, int64_t rows, int64_t len, int64_t k,
                              bool largest, uint32_t* values, int32_t* indices, void* scratch,
                              void* ws, hipStream_t stream) {
    using TV = RowTile<uint32_t, G, true>;
    using TU = RowTile<uint32_t, G, false>;
    static_assert(TV::kElems == TU::kElems, "one tile size per geometry");
    const uint32_t segs = (uint32_t)((len + TV::kElems - 1) / TV::kElems);
    const uint32_t nt = (uint32_t)(rows * segs);
    const unsigned threads = vec ? TV::kThreads : TU::kThreads;
    char* w = reinterpret_cast<char*>(ws);
    const TopkLayout l = topk_layout(rows, len, k);
    uint32_t* hist = reinterpret_cast<uint32_t*>(w + l.hist);
    uint64_t* state = reinterpret_cast<uint64_t*>(w + l.state);
    uint64_t* gather = reinterpret_cast<uint64_t*>(w + l.gather);
    uint32_t* offs = reinterpret_cast<uint32_t*>(w + l.offs);
    uint64_t* cand = reinterpret_cast<uint64_t*>(scratch);
    const uint32_t kk = (uint32_t)k, cap = topk_cap(len);
    if (segs > kTopkGatherSegs) return hipErrorInvalidValue;  // not on this route
    hipLaunchKernelGGL((vec ? k_topk_count0<TV, true> : k_topk_count0<TU, false>), dim3(nt),
                       dim3(threads), 0, stream, x, len, segs, largest, hist);
    uint32_t* rowhist = reinterpret_cast<uint32_t*>(w + l.rowhist);
    hipLaunchKernelGGL(k_topk_bucket, dim3((uint32_t)rows), dim3(kTopkDigits), 0, stream,
                       (const uint32_t*)hist, segs, kk, state, gather, offs, rowhist);
    hipLaunchKernelGGL((vec ? k_topk_gather<TV, true> : k_topk_gather<TU, false>), dim3(nt),
                       dim3(threads), 0, stream, x, len, segs, largest, (const uint64_t*)state,
                       (const uint64_t*)gather, (const uint32_t*)offs, cand, cap);
    // the LDS sort sized to the row (cap <= CAP)
    auto kf = cap > 8192 ? k_topk_finish<kTopkCand, false>
                         : (cap > 2048 ? k_topk_finish<8192, false> : k_topk_finish<2048, false>);
    hipLaunchKernelGGL(kf, dim3((uint32_t)rows * topk_parts(kk)), dim3(kTopkFinishThreads), 0,
                       stream, x, len, kk, largest, (const uint64_t*)state,
                       (const uint64_t*)gather, (const uint64_t*)cand, cap, segs,
                       (const uint32_t*)nullptr, (const uint32_t*)rowhist, values, indices);
    return hipGetLastError();
}

template <class G>
static hipError_t topk_tiles(bool vec, const uint32_t* x, int64_t rows, int64_t len, int64_t k,
                             bool largest, uint32_t* values, int32_t* indices, void* scratch,
                             void* ws, hipStream_t stream) {
    using TV = RowTile<uint32_t, G, true>;
    using TU = RowTile<uint32_t, G, false>;
    static_assert(TV::kElems == TU::kElems, "one tile size per geometry");
    const uint32_t segs = (uint32_t)((len + TV::kElems - 1) / TV::kElems);
    const uint32_t nt = (uint32_t)(rows * segs);
    const unsigned threads = vec ? TV::kThreads : TU::kThreads;
    const TopkLayout l = topk_layout(rows, len, k);
    uint32_t* tcount = reinterpret_cast<uint32_t*>(reinterpret_cast<char*>(ws) + l.offs);
    uint64_t* cand = reinterpret_cast<uint64_t*>(scratch);
    const uint32_t kk = (uint32_t)k;
    // every candidate in the finisher's LDS, every tile list on one slot per
    // finisher thread (CAP / kTopkFinishThreads of them)
    const uint32_t cap = (uint32_t)(len < (int64_t)segs * kTopkTileSlots
                                        ? len : (int64_t)segs * kTopkTileSlots);
    const uint32_t fcap = cap > 8192 ? kTopkCand : (cap > 2048 ? 8192 : 2048);
    if (segs != topk_tiles_segs(len) || segs > kTopkGatherSegs ||
        segs > fcap / kTopkFinishThreads)
        return hipErrorInvalidValue;  // not on this route
    hipLaunchKernelGGL((vec ? k_topk_tilesel<TV, true> : k_topk_tilesel<TU, false>), dim3(nt),
                       dim3(threads), 0, stream, x, len, segs, kk, largest, cand, tcount);
    auto kf = fcap == kTopkCand ? k_topk_finish<kTopkCand, true>
                                : (fcap == 8192 ? k_topk_finish<8192, true>
                                                : k_topk_finish<2048, true>);
    hipLaunchKernelGGL(kf, dim3((uint32_t)rows), dim3(kTopkFinishThreads), 0, stream, x, len, kk,
                       largest, (const uint64_t*)nullptr, (const uint64_t*)nullptr,
                       (const uint64_t*)cand, cap, segs, (const uint32_t*)tcount,
                       (const uint32_t*)nullptr, values, indices);
    return hipGetLastError();
}

hipError_t launch_topk(const float* x, float* values, int32_t* indices, int64_t rows, int64_t len,
                       int64_t k, bool largest, void* scratch, void* ws, hipStream_t stream) {
    if (rows == 0 || k == 0) return hipSuccess;
    const bool vec = (len % 4 == 0) && ((uintptr_t)x % 16) == 0;
    if (topk_tiles_route(len, k)) {
        const uint32_t* xb = reinterpret_cast<const uint32_t*>(x);
        uint32_t* vb = reinterpret_cast<uint32_t*>(values);
        return topk_gather_tile(len) == 8192
                   ? topk_tiles<RGeomM>(vec, xb, rows, len, k, largest, vb, indices, scratch, ws,
                                        stream)
                   : topk_tiles<RGeomS>(vec, xb, rows, len, k, largest, vb, indices, scratch, ws,
                                        stream);
    }
    if (topk_gather_route(len, k)) {
        const uint32_t* xb = reinterpret_cast<const uint32_t*>(x);
        uint32_t* vb = reinterpret_cast<uint32_t*>(values);
        return topk_gather_tile(len) == 8192
                   ? topk_gather<RGeomM>(vec, xb, rows, len, k, largest, vb, indices, scratch, ws,
                                         stream)
                   : topk_gather<RGeomS>(vec, xb, rows, len, k, largest, vb, indices, scratch, ws,
                                         stream);
    }
    const size_t mb = align256((size_t)rows * (size_t)k * 4);
    char* s = reinterpret_cast<char*>(scratch);
    uint32_t* sel_vals = reinterpret_cast<uint32_t*>(s);
    int32_t* sel_idx = reinterpret_cast<int32_t*>(s + mb);
    const uint32_t* xb = reinterpret_cast<const uint32_t*>(x);
    const int64_t t = row_tile(len);
    hipError_t e;
    if (t == 32768)
        e = topk_select<RGeomL>(vec, xb, rows, len, k, largest, sel_vals, sel_idx, ws, stream);
    else if (t == 8192)
        e = topk_select<RGeomM>(vec, xb, rows, len, k, largest, sel_vals, sel_idx, ws, stream);
    else
        e = topk_select<RGeomS>(vec, xb, rows, len, k, largest, sel_vals, sel_idx, ws, stream);
    if (e != hipSuccess) return e;
    if (k <= kTopkSortMax) {
        uint32_t npow = 1;
        while (npow < (uint32_t)k) npow <<= 1;
        hipLaunchKernelGGL(k_topk_sort, dim3((uint32_t)rows), dim3(kTopkSortThreads), 0, stream,
                           (const uint32_t*)sel_vals, (const int32_t*)sel_idx,
                           reinterpret_cast<uint32_t*>(values), indices, (uint32_t)k, npow,
                           largest);
        return hipGetLastError();
    }
    // the kept elements in order: a stable sort of each row's k values,
    // carrying their indices (ties keep index order, as the split left them)
    return launch_radix_sort_typed(KeyType::F32, largest, sel_vals, values, sel_idx, indices,
                                   s + 2 * mb, reinterpret_cast<int32_t*>(s + 3 * mb), rows, k,
                                   ws, topk_ws_bytes(rows, len, k), stream);
}

}  // namespace ls
