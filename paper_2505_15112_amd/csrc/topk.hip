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
// No workgroup waits for another during the histogram rounds: each tile
// writes its 256 digit counts to its own slots, and the row's last tile to
// arrive (the per-row arrival counter of the row kernels) adds them and
// picks the bucket.  The split is a two-chain decoupled look-back (elements
// above T, elements equal to T), so the output keeps index order.
#include <limits.h>

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
    for (uint32_t size = 2; size <= npow; size <<= 1) {
        for (uint32_t stride = size >> 1; stride > 0; stride >>= 1) {
            for (uint32_t t = threadIdx.x; t < npow / 2; t += kTopkSortThreads) {
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
    for (uint32_t i = threadIdx.x; i < k; i += kTopkSortThreads) {
        const uint64_t c = s[i];
        const uint32_t key = (uint32_t)(c >> 32);
        const uint32_t code = largest ? key : ~key;
        values[row * k + i] = code ^ ((code >> 31) ? 0x80000000u : 0xFFFFFFFFu);
        indices[row * k + i] = (int32_t)~(uint32_t)c;
    }
}

// ---------------------------------------------------------------- launch

// Workspace: header | two look-back chains (rows x segments words each) |
// digit counts (rows x segments x 256) | row states (2 words) | arrival
// counters; the final radix sort (k > kTopkSortMax) reuses the front.
// Scratch: the k kept values and indices per row, and for the radix sort its
// two ping-pong buffers.
static size_t align256(size_t b) { return (b + 255) / 256 * 256; }
struct TopkLayout {
    size_t hist, state, arrivals, end;
};
static TopkLayout topk_layout(int64_t rows, int64_t len) {
    const size_t tiles = (size_t)rows * (size_t)row_segments(len);
    TopkLayout l;
    l.hist = align256(kWsHeader + 2 * tiles * sizeof(uint64_t));
    l.state = align256(l.hist + tiles * kTopkDigits * sizeof(uint32_t));
    l.arrivals = l.state + (size_t)rows * 2 * sizeof(uint64_t);
    l.end = l.arrivals + (size_t)rows * sizeof(uint64_t);
    return l;
}
size_t topk_ws_bytes(int64_t rows, int64_t len, int64_t k) {
    const size_t a = topk_layout(rows, len).end;
    const size_t b = k > kTopkSortMax ? radix_rows_ws_bytes(rows, k) : 0;
    return a > b ? a : b;
}
size_t topk_scratch_bytes(int64_t rows, int64_t k) {
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
    const TopkLayout l = topk_layout(rows, len);
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

hipError_t launch_topk(const float* x, float* values, int32_t* indices, int64_t rows, int64_t len,
                       int64_t k, bool largest, void* scratch, void* ws, hipStream_t stream) {
    if (rows == 0 || k == 0) return hipSuccess;
    const bool vec = (len % 4 == 0) && ((uintptr_t)x % 16) == 0;
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
