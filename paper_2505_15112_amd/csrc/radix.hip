// radix.hip -- least-significant-digit radix sort of uint32 keys with a
// stable permutation (Section 5 "Radix Sort": a loop over the bits from the
// least significant one, each step a stable split; Section 6 returns the
// indices as PyTorch's sort() does).
//
//  * 1 bit per pass: one pre-pass reads the keys once and builds the 8 x 16
//    histogram of all 4-bit digits (per-block partial histograms, then one
//    block adds them); then 32 split passes (compact.hip's split kernel with
//    the flag "bit b is 0"), the number of zero bits of pass b read off the
//    histogram, so no pass needs its own counting kernel.
//  * 4 bits per pass: 8 passes, each three kernels with no inter-workgroup
//    waiting: every tile counts its 16 digits (keys read once more), the
//    digit-major count table (16 x tiles) is turned into output offsets by
//    one exclusive 1-D scan (scan1d's look-back kernel: the offset of digit d
//    in tile t is the number of keys with a smaller digit, plus those with
//    digit d in earlier tiles), and
//    every tile ranks its keys per digit with a wavefront multi-split (one
//    ballot per digit bit; the lanes holding the same digit are the AND of
//    the matching ballots, the rank is the count of them below the lane),
//    sorts them by digit in LDS and writes each digit's run contiguously.
//    (A single-pass version carrying the 16 counts by a 16-chain decoupled
//    look-back measured 2x slower per pass on MI355X: every tile's walk
//    waited on its predecessors' 16 words.)
//  * 8 bits per pass: 4 passes of the same three kernels with 256 digits;
//    ranking goes through per-wave digit counts in LDS (see below).  Half the
//    passes of the 4-bit sort, so half its key and index traffic.
// All variants give identical output: a stable sort is unique.
#include "launch.hpp"
#include "tile.hpp"

namespace ls {

constexpr int kHistWords = 8 * 16;  // final counts, one 64-bit word each, after the header
constexpr size_t kRadixStatusOffset = kWsHeader + kHistWords * sizeof(uint64_t);
constexpr int kHistBlocks = 512;  // blocks of the histogram pre-pass (one partial each)

constexpr int kR4Waves = 8;
constexpr int kR4Chunks = 16;  // 64 keys (one per lane) per chunk
constexpr int64_t kR4Tile = kR4Waves * kR4Chunks * kWave;  // 8192 keys
constexpr int64_t kR1Tile = 4096;  // at most compact.hip's split tile: enough status words

static inline int64_t r4_tiles(int64_t n) { return (n + kR4Tile - 1) / kR4Tile; }

// ---------------------------------------------------------------- histogram

// 16 copies of the 8 x 16 histogram in LDS, the copy picked by lane & 15 and
// held in the low address bits: the lanes of one atomic instruction rarely
// hit the same word, and spread over the banks.
constexpr int kHistCopies = 16;

__device__ __forceinline__ void hist_add(uint32_t* s_h, uint32_t k, uint32_t copy) {
#pragma unroll
    for (int p = 0; p < 8; ++p)
        atomicAdd(&s_h[(p * 16 + ((k >> (4 * p)) & 15u)) * kHistCopies + copy], 1u);
}

__global__ __launch_bounds__(256) void k_digit_hist(const uint32_t* keys, int64_t n, bool vec,
                                                    uint32_t* part) {
    __shared__ uint32_t s_h[kHistWords * kHistCopies];
    for (int i = threadIdx.x; i < kHistWords * kHistCopies; i += blockDim.x) s_h[i] = 0;
    __syncthreads();
    const uint32_t copy = threadIdx.x & (kHistCopies - 1);
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t t0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int64_t done = 0;
    if (vec) {  // 4 keys per 16-byte load, 4 loads in flight per thread
        const u32x4* k4 = reinterpret_cast<const u32x4*>(keys);
        const int64_t n4 = n / 4;
        for (int64_t i = t0; i < n4; i += 4 * stride) {
            u32x4 v[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int64_t q = i + u * stride;
                v[u] = q < n4 ? k4[q] : u32x4{0, 0, 0, 0};
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                if (i + u * stride < n4) {
                    hist_add(s_h, v[u].x, copy);
                    hist_add(s_h, v[u].y, copy);
                    hist_add(s_h, v[u].z, copy);
                    hist_add(s_h, v[u].w, copy);
                }
            }
        }
        done = n4 * 4;
    }
    for (int64_t i = done + t0; i < n; i += stride) hist_add(s_h, keys[i], copy);
    __syncthreads();
    if (threadIdx.x < kHistWords) {
        uint32_t c = 0;
#pragma unroll
        for (int k = 0; k < kHistCopies; ++k) c += s_h[threadIdx.x * kHistCopies + k];
        part[blockIdx.x * kHistWords + threadIdx.x] = c;
    }
}

// One block adds the per-block histograms into the final 128 counts.
__global__ __launch_bounds__(1024) void k_hist_reduce(const uint32_t* part, int nblocks,
                                                      uint64_t* hist) {
    __shared__ uint32_t s_sum[8][kHistWords];
    const int word = threadIdx.x % kHistWords, slice = threadIdx.x / kHistWords;  // 8 slices
    uint32_t c = 0;
    for (int b = slice; b < nblocks; b += 8) c += part[b * kHistWords + word];
    s_sum[slice][word] = c;
    __syncthreads();
    if (threadIdx.x < kHistWords) {
        uint32_t t = 0;
#pragma unroll
        for (int k = 0; k < 8; ++k) t += s_sum[k][threadIdx.x];
        hist[threadIdx.x] = t;
    }
}

// The scatter kernels have no inter-workgroup order, so their tile index is
// free: workgroups are dealt to the 8 XCDs round-robin by block index, and
// this gives each XCD one contiguous range of tiles.  Neighbouring tiles then
// write the two halves of the cache lines at their shared run boundaries from
// the same L2, where the partial lines merge before going to HBM.  (A
// bijection on block indices whatever the placement; only speed depends on
// the round-robin dealing.)
constexpr uint32_t kXcds = 8;
__device__ __forceinline__ uint32_t xcd_tile(uint32_t b, uint32_t nblocks) {
    const uint32_t x = b % kXcds, k = b / kXcds;
    const uint32_t per = nblocks / kXcds, extra = nblocks % kXcds;
    return x * per + (x < extra ? x : extra) + k;
}

// ---------------------------------------------------------------- 4-bit pass

// Lanes whose digit equals `d`, from the four digit-bit ballots and the
// ballot of valid lanes.
__device__ __forceinline__ uint64_t digit_lanes(uint32_t d, uint64_t valid, uint64_t b0,
                                                uint64_t b1, uint64_t b2, uint64_t b3) {
    return valid & ((d & 1) ? b0 : ~b0) & ((d & 2) ? b1 : ~b1) & ((d & 4) ? b2 : ~b2) &
           ((d & 8) ? b3 : ~b3);
}

__device__ __forceinline__ uint32_t lanes_below(uint64_t m) {
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
}

__device__ __forceinline__ uint32_t lane_shfl(uint32_t v, int src_lane) {
    return (uint32_t)__builtin_amdgcn_ds_bpermute(src_lane << 2, (int)v);
}

// A wave's chunks of 64 source indices straight into LDS, chunk j at
// lds + 64 j: the immediate offset of an LDS-direct load is added to the
// global and to the LDS address alike, so one address pair serves them all.
// The scatters read keys and indices once, nontemporally (cache policy bit
// "nt" of the LDS-direct load); measured 3-9 % faster sorts than cached loads.
constexpr int kLoadNT = 2;
template <int... J>
__device__ __forceinline__ void indices_to_lds(const int32_t* lane_src, int32_t* lds,
                                               std::integer_sequence<int, J...>) {
    (__builtin_amdgcn_global_load_lds((const void*)lane_src, lds, 4, J * kWave * 4, kLoadNT), ...);
}

// Per-tile digit counts: counts[d * ntiles + tile] (digit-major, so the
// spine kernel scans contiguous columns).  Order does not matter here, so the
// keys are read with 16-byte loads when aligned.
__global__ __launch_bounds__(kR4Waves* kWave) LS_OCCUPANCY4 void k_radix4_count(const uint32_t* keys, int64_t n,
                                                                  int shift, bool vec,
                                                                  uint32_t* counts,
                                                                  uint32_t ntiles) {
    __shared__ uint32_t s_cnt[kR4Waves][16];
    const int lane = lane_id();
    const int w = threadIdx.x / kWave;
    // tiles dealt XCD-aware, as in the scatter: neighbouring tiles' count words
    // share cache lines, which then merge in one L2
    const uint32_t tile = xcd_tile(blockIdx.x, gridDim.x);
    const int64_t tbase = (int64_t)tile * kR4Tile;
    const bool full = tbase + kR4Tile <= n;
    uint32_t run = 0;  // lane L < 16: this wave's count of digit L
    // every lane holds a key: the lanes holding digit lane & 15 are the AND
    // over the digit bits of ballot ^ el (el: all ones where lane & 15 has
    // the bit clear), ballots first (see digit4_masks)
    uint32_t el[4];
#pragma unroll
    for (int b = 0; b < 4; ++b) {
        el[b] = (uint32_t)__builtin_amdgcn_sbfe((int)~(uint32_t)lane, b, 1);
        asm("" : "+v"(el[b]));
    }
    auto count64_all = [&](uint32_t key) {
        const uint32_t d = (key >> shift) & 15u;
        uint64_t bb[4];
#pragma unroll
        for (int b = 0; b < 4; ++b) bb[b] = __ballot((d >> b) & 1u);
        uint32_t lo = ~0u, hi = ~0u;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            lo &= (uint32_t)bb[b] ^ el[b];
            hi &= (uint32_t)(bb[b] >> 32) ^ el[b];
            asm("" : "+v"(lo), "+v"(hi));
        }
        run += (uint32_t)__builtin_popcount(lo) + (uint32_t)__builtin_popcount(hi);
    };
    auto count64 = [&](uint32_t key, bool ok) {
        const uint32_t d = (key >> shift) & 15u;
        const uint64_t valid = __ballot(ok);
        const uint64_t b0 = __ballot(ok && (d & 1));
        const uint64_t b1 = __ballot(ok && (d & 2));
        const uint64_t b2 = __ballot(ok && (d & 4));
        const uint64_t b3 = __ballot(ok && (d & 8));
        run += (uint32_t)__builtin_popcountll(digit_lanes((uint32_t)(lane & 15), valid, b0, b1, b2, b3));
    };
    if (vec && full) {  // this wave's 1024 keys as 4 x 16-byte loads per lane
        const u32x4* k4 = reinterpret_cast<const u32x4*>(keys + tbase + (int64_t)w * kR4Chunks * kWave);
        u32x4 v[kR4Chunks / 4];
#pragma unroll
        for (int j = 0; j < kR4Chunks / 4; ++j) v[j] = k4[j * kWave + lane];
#pragma unroll
        for (int j = 0; j < kR4Chunks / 4; ++j) {
            count64_all(v[j].x);
            count64_all(v[j].y);
            count64_all(v[j].z);
            count64_all(v[j].w);
        }
    } else {
        const int64_t wbase = tbase + (int64_t)w * kR4Chunks * kWave;
#pragma unroll
        for (int j = 0; j < kR4Chunks; ++j) {
            const int64_t i = wbase + j * kWave + lane;
            const bool ok = i < n;
            count64(ok ? keys[i] : 0u, ok);
        }
    }
    if (lane < 16) s_cnt[w][lane] = run;
    __syncthreads();
    if (threadIdx.x < 16) {
        uint32_t t = 0;
#pragma unroll
        for (int k = 0; k < kR4Waves; ++k) t += s_cnt[k][threadIdx.x];
        counts[(int64_t)threadIdx.x * ntiles + tile] = t;
    }
}

// Peer masks of a 4-bit digit when every lane of the wave holds a key: the
// lanes whose digit equals this lane's digit d (`same`) and the lanes whose
// digit equals this lane's number mod 16 (`of_lane`, for the chunk's count of
// that digit).  Per digit bit b: the ballot of the lanes with the bit set,
// and m &= ballot ^ e with e all ones where the wanted digit has the bit
// clear (ne: this lane's digit, el: its lane number's, a sign-extended bit
// field of the complement).  All ballots first, so that no read of a ballot
// waits on its write; the empty asm statements only hide values from the
// optimiser (they emit nothing), which keeps each m &= ballot ^ e one
// three-input bit operation.
__device__ __forceinline__ void digit4_masks(uint32_t d, const uint32_t (&el)[4], uint64_t& same,
                                             uint64_t& of_lane) {
    const int nd = (int)~d;
    uint32_t ne[4];
    uint64_t bb[4];
#pragma unroll
    for (int b = 0; b < 4; ++b) {
        ne[b] = (uint32_t)__builtin_amdgcn_sbfe(nd, b, 1);
        asm("" : "+v"(ne[b]));
    }
#pragma unroll
    for (int b = 0; b < 4; ++b) bb[b] = __ballot(ne[b] == 0u);
    uint32_t slo = ~0u, shi = ~0u, llo = ~0u, lhi = ~0u;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
        slo &= (uint32_t)bb[b] ^ ne[b];
        shi &= (uint32_t)(bb[b] >> 32) ^ ne[b];
        llo &= (uint32_t)bb[b] ^ el[b];
        lhi &= (uint32_t)(bb[b] >> 32) ^ el[b];
        asm("" : "+v"(slo), "+v"(shi), "+v"(llo), "+v"(lhi));
    }
    same = ((uint64_t)shi << 32) | slo;
    of_lane = ((uint64_t)lhi << 32) | llo;
}

// Rank and scatter one tile of 8192 keys (one key per lane per chunk, so the
// chunk's index order is the lane order) with the offsets from the spine.
template <bool HAS_PERM_IN, bool WITH_PERM>
__global__ __launch_bounds__(kR4Waves* kWave) LS_OCCUPANCY4 void k_radix4_scatter(
    const uint32_t* keys_in, const int32_t* perm_in, uint32_t* keys_out, int32_t* perm_out,
    int64_t n, int shift, uint32_t* offsets, uint32_t ntiles) {
    __shared__ uint32_t s_cnt[kR4Waves][16];
    __shared__ uint32_t s_tstart[16];  // first slot of digit d in the tile's digit order
    __shared__ uint32_t s_off[16];     // global position minus tile slot, per digit
    __shared__ uint32_t s_stage[kR4Tile];
    // the tile's source indices, loaded straight into LDS at the start (in
    // the tile's index order) so that they cost no registers while ranking
    __shared__ int32_t s_pin[WITH_PERM && HAS_PERM_IN ? kR4Tile : 1];

    const int64_t tile = xcd_tile(blockIdx.x, gridDim.x);
    const int lane = lane_id();
    const int w = threadIdx.x / kWave;
    const int64_t tbase = tile * kR4Tile;
    const int64_t wbase = tbase + (int64_t)w * kR4Chunks * kWave;
    const bool full = tbase + kR4Tile <= n;
    const uint32_t valid = full ? (uint32_t)kR4Tile : (uint32_t)(n - tbase);

    uint32_t gbase = 0;  // lane d < 16 of wave 0: global position of the tile's first digit-d key
    if (threadIdx.x < 16) {
        uint32_t* o = offsets + (int64_t)threadIdx.x * ntiles + tile;
        gbase = *o;
        *o = 0;  // offsets can reach 2^30 and more: leave the workspace word zero
    }

    // The tile body, compiled twice: for full tiles (every lane holds a key,
    // no per-lane bounds) and for the last, ragged tile.
    auto body = [&](auto full_c) {
        constexpr bool FULL = decltype(full_c)::value;
        auto in_range = [&](int j) { return FULL || wbase + j * kWave + lane < n; };
        const uint32_t* kw = keys_in + wbase;
        // Source indices first, straight into LDS; lanes past the end load
        // nothing and their slots are never read.
        if (WITH_PERM && HAS_PERM_IN) {
            const int32_t* pw = perm_in + wbase;
            int32_t* lw = s_pin + w * kR4Chunks * kWave;
            if (FULL) {
                indices_to_lds(pw + lane, lw, std::make_integer_sequence<int, kR4Chunks>{});
            } else {
#pragma unroll
                for (int j = 0; j < kR4Chunks; ++j)
                    if (in_range(j))
                        __builtin_amdgcn_global_load_lds((const void*)(pw + j * kWave + lane),
                                                         lw + j * kWave, 4, 0, 0);
            }
        }
        uint32_t key[kR4Chunks];
#pragma unroll
        for (int j = 0; j < kR4Chunks; ++j)
            key[j] = in_range(j) ? __builtin_nontemporal_load(&kw[j * kWave + lane]) : 0u;

        // Per-chunk digit counts first (independent), then the stable rank of
        // each key: its digit's count in the wave's earlier chunks plus the
        // lanes below it holding the same digit.
        uint32_t cnt[kR4Chunks];
        uint32_t rank[kR4Chunks];
        if (FULL) {
            uint32_t el[4];
#pragma unroll
            for (int b = 0; b < 4; ++b) {
                el[b] = (uint32_t)__builtin_amdgcn_sbfe((int)~(uint32_t)lane, b, 1);
                asm("" : "+v"(el[b]));
            }
#pragma unroll
            for (int j = 0; j < kR4Chunks; ++j) {
                uint64_t same, of_lane;
                digit4_masks((key[j] >> shift) & 15u, el, same, of_lane);
                rank[j] = lanes_below(same);
                cnt[j] = (uint32_t)__builtin_popcountll(of_lane);
            }
        } else {
#pragma unroll
            for (int j = 0; j < kR4Chunks; ++j) {
                const bool ok = in_range(j);
                const uint32_t d = (key[j] >> shift) & 15u;
                const uint64_t valid_l = __ballot(ok);
                const uint64_t b0 = __ballot(ok && (d & 1));
                const uint64_t b1 = __ballot(ok && (d & 2));
                const uint64_t b2 = __ballot(ok && (d & 4));
                const uint64_t b3 = __ballot(ok && (d & 8));
                rank[j] = lanes_below(digit_lanes(d, valid_l, b0, b1, b2, b3));
                cnt[j] = (uint32_t)__builtin_popcountll(
                    digit_lanes((uint32_t)(lane & 15), valid_l, b0, b1, b2, b3));
            }
        }
        uint32_t run = 0;
#pragma unroll
        for (int j = 0; j < kR4Chunks; ++j) {
            const uint32_t d = (key[j] >> shift) & 15u;
            rank[j] += lane_shfl(run, (int)d);
            run += cnt[j];
        }
        if (lane < 16) s_cnt[w][lane] = run;
        // the index loads were issued first: long done, and no stores yet
        if (WITH_PERM && HAS_PERM_IN) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();

        // lanes 0..15: count of digit `lane` in earlier waves, and the tile total
        uint32_t wofs = 0, tot = 0;
#pragma unroll
        for (int k = 0; k < kR4Waves; ++k) {
            const uint32_t c = s_cnt[k][lane & 15];
            if (k < w) wofs += c;
            tot += c;
        }
        if (w == 0) {
            const uint32_t t16 = lane < 16 ? tot : 0u;
            const uint32_t tstart = wave_incl_scan(t16) - t16;
            if (lane < 16) {
                s_tstart[lane] = tstart;
                s_off[lane] = gbase - tstart;
            }
        }
        __syncthreads();

        // Sort the tile by digit in LDS (slot = digit start + earlier waves +
        // rank), then write each digit's run with consecutive threads.
        const uint32_t wstart = (lane < 16 ? s_tstart[lane] : 0u) + wofs;  // lane d: this wave's slot 0 for d
        uint32_t slot[kR4Chunks];
#pragma unroll
        for (int j = 0; j < kR4Chunks; ++j) {
            const uint32_t d = (key[j] >> shift) & 15u;
            slot[j] = lane_shfl(wstart, (int)d) + rank[j];
            if (FULL || (in_range(j) && slot[j] < kR4Tile)) s_stage[slot[j]] = key[j];
        }
        __syncthreads();
        // All staged keys, then their positions, then the stores.  A position
        // is clamped to the array (it is inside always; the clamp keeps a
        // corrupted offsets table from writing out of bounds).
        const uint32_t last = (uint32_t)(n - 1);  // n <= INT32_MAX
        uint32_t sk[kR4Chunks], pos[kR4Chunks];
#pragma unroll
        for (int j = 0; j < kR4Chunks; ++j) sk[j] = s_stage[threadIdx.x + j * kR4Waves * kWave];
#pragma unroll
        for (int j = 0; j < kR4Chunks; ++j)
            pos[j] = min(s_off[(sk[j] >> shift) & 15u] + (uint32_t)threadIdx.x + j * kR4Waves * kWave,
                         last);
#pragma unroll
        for (int j = 0; j < kR4Chunks; ++j)
            if (FULL || threadIdx.x + j * kR4Waves * kWave < valid) keys_out[pos[j]] = sk[j];
        if (WITH_PERM) {
            __syncthreads();
#pragma unroll
            for (int j = 0; j < kR4Chunks; ++j) {
                const int32_t pv = HAS_PERM_IN ? s_pin[(w * kR4Chunks + j) * kWave + lane]
                                               : (int32_t)(wbase + j * kWave + lane);
                if (FULL || (in_range(j) && slot[j] < kR4Tile)) s_stage[slot[j]] = (uint32_t)pv;
            }
            __syncthreads();
#pragma unroll
            for (int j = 0; j < kR4Chunks; ++j) sk[j] = s_stage[threadIdx.x + j * kR4Waves * kWave];
#pragma unroll
            for (int j = 0; j < kR4Chunks; ++j)
                if (FULL || threadIdx.x + j * kR4Waves * kWave < valid)
                    perm_out[pos[j]] = (int32_t)sk[j];
        }
    };
    if (full)
        body(std::true_type{});
    else
        body(std::false_type{});
}

// ---------------------------------------------------------------- key codes

// Signed and floating-point keys sort as unsigned integers after an encoding
// (Section 5 "Radix Sort": invert the most significant bit of non-negative
// numbers and every bit of negative ones; signed integers only need the
// most significant bit inverted), and are decoded when the last pass writes
// them.  Descending order inverts every bit of the code as well.  The first
// pass applies `code` on its loads, the last pass `decode` on its stores;
// every other pass (and the plain unsigned sort) uses the identity.
struct KeyCode {
    uint32_t pos, neg;  // code(k) = k ^ (sign bit of k ? neg : pos)
    int top;            // sign bit position: 31 (32-bit keys) or 15 (16-bit)
    __device__ uint32_t apply(uint32_t k) const { return k ^ (((k >> top) & 1u) ? neg : pos); }
};
struct KeyDecode {
    uint32_t pre, one, zero;  // e' = e ^ pre; k = e' ^ (bit top of e' ? one : zero)
    int top;
    __device__ uint32_t apply(uint32_t e) const {
        e ^= pre;
        return e ^ (((e >> top) & 1u) ? one : zero);
    }
};

// ---------------------------------------------------------------- 8-bit pass

// 4 passes of 8-bit digits: the same count -> scan -> scatter structure as the
// 4-bit pass, with 256 digits.  Ranking cannot give every digit a lane, so
// each wave keeps its digit counts in LDS: per chunk of 64 keys, the lanes
// holding one digit (found with 8 ballots) are a peer group, the group's
// lowest lane adds the group size to the wave's count of that digit (one LDS
// add per group, never two lanes on one word), every lane reads the count
// back, and a key's rank is that count minus the group size plus its peers
// in lower lanes.  A wave's LDS operations execute in issue order, so ranks
// follow the index order.
constexpr int kR8Waves = 8;
constexpr int kR8Chunks = 16;
constexpr int64_t kR8Tile = kR8Waves * kR8Chunks * kWave;  // 8192 keys
constexpr int kR8Digits = 256;


// Lanes holding the same 8-bit digit as this lane, when every lane of the
// wave holds a key: the AND over the digit bits of that bit's ballot,
// complemented where this lane's bit is 0.  Per bit: e = all ones if the bit
// is 0 (a sign-extended bit field of ~d), the ballot of e == 0, and
// m &= ballot ^ e for each 32-bit half.  The empty asm statements only hide
// values from the optimiser (they emit nothing): the ballot then stays a
// test of e, and each m &= ballot ^ e stays one three-input bit operation
// instead of being regrouped with the next bit into more operations.
__device__ __forceinline__ uint64_t peers8_all(uint32_t d) {
    const int nd = (int)~d;
    uint32_t e[8];
    uint64_t bb[8];
#pragma unroll
    for (int b = 0; b < 8; ++b) {
        e[b] = (uint32_t)__builtin_amdgcn_sbfe(nd, b, 1);
        asm("" : "+v"(e[b]));
    }
    // all ballots first: each is read well after it is written, so no wait
    // states go in between
#pragma unroll
    for (int b = 0; b < 8; ++b) bb[b] = __ballot(e[b] == 0u);
    uint32_t lo = ~0u, hi = ~0u;
#pragma unroll
    for (int b = 0; b < 8; ++b) {
        lo &= (uint32_t)bb[b] ^ e[b];
        hi &= (uint32_t)(bb[b] >> 32) ^ e[b];
        asm("" : "+v"(lo), "+v"(hi));
    }
    return ((uint64_t)hi << 32) | lo;
}

// The same among the `ok` lanes (a ragged tile).
__device__ __forceinline__ uint64_t peers8(uint32_t d, bool ok) {
    uint64_t m = __ballot(ok);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
        const uint64_t bb = __ballot(ok && ((d >> b) & 1u));
        m &= ((d >> b) & 1u) ? bb : ~bb;
    }
    return m;
}

// Per-tile counts of the 256 digits.  Keys form rows of `len` (one row of n
// for a 1-D sort; tiles never straddle rows, tpr tiles per row), and the count
// of digit d in tile tr of row r goes to counts[(r * 256 + d) * tpr + tr]: per
// row digit-major, so that one exclusive scan per row turns the table into
// each (digit, tile)'s first output position in the row.  Order does not
// matter here: keys are read with 16-byte loads when aligned and counted
// with plain LDS atomics, into 4 histograms per wave (picked by lane & 3) so
// that equal digits in one instruction collide at most 16 ways.
constexpr int kR8Sub = 4;
template <class K>
__global__ __launch_bounds__(kR8Waves* kWave) LS_OCCUPANCY4 void k_radix8_count(
    const K* keys, int64_t len, uint32_t tpr, int shift, bool vec, uint32_t* counts,
    KeyCode code) {
    __shared__ uint32_t s_h[kR8Waves * kR8Sub][kR8Digits];
    const int lane = lane_id();
    const int w = threadIdx.x / kWave;
    uint32_t* h = s_h[w * kR8Sub + (lane & (kR8Sub - 1))];
    // tiles dealt XCD-aware, as in the scatter: neighbouring tiles' count words
    // share cache lines, which then merge in one L2 (dealt round-robin by
    // block index they went to HBM as 8x the table's bytes)
    const uint32_t tile = xcd_tile(blockIdx.x, gridDim.x);
    const uint32_t row = tile / tpr, tr = tile - row * tpr;
    const int64_t tstart = (int64_t)tr * kR8Tile;  // within the row
    const K* kr = keys + (int64_t)row * len;
    const int64_t wbase = tstart + (int64_t)w * kR8Chunks * kWave;
    const bool fast = vec && tstart + kR8Tile <= len;
    // The key loads first: clearing the histograms runs under their latency.
    // Fast path: 16-byte loads, 4 of 32-bit keys or 8 of 16-bit keys each.
    constexpr int kPer = 16 / (int)sizeof(K);
    constexpr int kLoads = kR8Chunks / kPer;
    u32x4 v[kLoads];
    uint32_t k[kR8Chunks];
    if (fast) {
        const u32x4* k4 = reinterpret_cast<const u32x4*>(kr + wbase);
#pragma unroll
        for (int j = 0; j < kLoads; ++j) v[j] = k4[j * kWave + lane];
    } else {
#pragma unroll
        for (int j = 0; j < kR8Chunks; ++j) {
            const int64_t i = wbase + j * kWave + lane;
            k[j] = i < len ? (uint32_t)kr[i] : 0u;
        }
    }
    for (int i = threadIdx.x; i < kR8Waves * kR8Sub * kR8Digits; i += kR8Waves * kWave)
        (&s_h[0][0])[i] = 0;
    __syncthreads();
    // the key encoding (first pass of signed or float keys only) is left out
    // of the loop when it is the identity
    auto count_all = [&](auto coded_c) {
        constexpr bool CODED = decltype(coded_c)::value;
        auto enc = [&](uint32_t x) { return CODED ? code.apply(x) : x; };
        if (fast) {
#pragma unroll
            for (int j = 0; j < kLoads; ++j)
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const uint32_t word = v[j][c];
                    if (sizeof(K) == 4) {
                        atomicAdd(&h[(enc(word) >> shift) & 255u], 1u);
                    } else {
                        atomicAdd(&h[(enc(word & 0xFFFFu) >> shift) & 255u], 1u);
                        atomicAdd(&h[(enc(word >> 16) >> shift) & 255u], 1u);
                    }
                }
        } else {
#pragma unroll
            for (int j = 0; j < kR8Chunks; ++j)
                if (wbase + j * kWave + lane < len) atomicAdd(&h[(enc(k[j]) >> shift) & 255u], 1u);
        }
    };
    if (code.pos | code.neg)
        count_all(std::true_type{});
    else
        count_all(std::false_type{});
    __syncthreads();
    if (threadIdx.x < kR8Digits) {
        uint32_t t = 0;
#pragma unroll
        for (int q = 0; q < kR8Waves * kR8Sub; ++q) t += s_h[q][threadIdx.x];
        counts[((int64_t)row * kR8Digits + threadIdx.x) * tpr + tr] = t;
    }
}

// Rank and scatter one tile of 8192 keys (one key per lane per chunk, so the
// chunk's index order is the lane order) with the offsets from the scanned
// table; rows and tiles as in k_radix8_count, the permutation holding indices
// within the row.
template <class K, bool HAS_PERM_IN, bool WITH_PERM>
__global__ __launch_bounds__(kR8Waves* kWave) LS_OCCUPANCY4 void k_radix8_scatter(
    const K* keys_in, const int32_t* perm_in, K* keys_out, int32_t* perm_out, int64_t len,
    uint32_t tpr, int shift, uint32_t* offsets, KeyCode code, KeyDecode decode) {
    // per-wave digit counts during ranking, then each wave's first slot per digit
    __shared__ uint32_t s_wh[kR8Waves][kR8Digits];
    __shared__ uint32_t s_off[kR8Digits];  // global row position minus tile slot, per digit
    __shared__ uint32_t s_part[kR8Digits / kWave];
    __shared__ uint32_t s_stage[kR8Tile];
    // the tile's source indices, loaded straight into LDS at the start (in
    // the tile's index order) so that they arrive while the keys are ranked
    __shared__ int32_t s_pin[WITH_PERM && HAS_PERM_IN ? kR8Tile : 1];

    const uint32_t tile = xcd_tile(blockIdx.x, gridDim.x);
    const int lane = lane_id();
    const int w = threadIdx.x / kWave;
    const uint32_t row = tile / tpr, tr = tile - row * tpr;
    const int64_t rbase = (int64_t)row * len;
    const int64_t tstart = (int64_t)tr * kR8Tile;  // within the row
    const int64_t wbase = tstart + (int64_t)w * kR8Chunks * kWave;
    const bool full = tstart + kR8Tile <= len;
    const uint32_t valid = full ? (uint32_t)kR8Tile : (uint32_t)(len - tstart);
    const K* kw = keys_in + rbase + wbase;  // this wave's keys
    K* kout = keys_out + rbase;

    for (int i = threadIdx.x; i < kR8Waves * kR8Digits; i += kR8Waves * kWave) (&s_wh[0][0])[i] = 0;
    uint32_t gbase = 0;  // thread d < 256: global row position of the tile's first digit-d key
    if (threadIdx.x < kR8Digits) {
        uint32_t* o = offsets + ((int64_t)row * kR8Digits + threadIdx.x) * tpr + tr;
        gbase = *o;
        *o = 0;  // offsets can reach 2^30 and more: leave the workspace word zero
    }

    // The tile body, compiled twice: for full tiles (every lane holds a key,
    // no per-lane bounds) and for the ragged last tile of a row.
    auto body = [&](auto full_c) {
        constexpr bool FULL = decltype(full_c)::value;
        auto in_range = [&](int j) { return FULL || wbase + j * kWave + lane < len; };

        // Source indices first, straight into LDS (no registers: ranking
        // needs them), then the keys.  The LDS-direct load of a chunk writes
        // lane l's 4 bytes at the chunk's slot + 4 l; lanes past the end load
        // nothing and their slots are never read.
        if (WITH_PERM && HAS_PERM_IN) {
            const int32_t* pw = perm_in + rbase + wbase;
            int32_t* lw = s_pin + w * kR8Chunks * kWave;
            if (FULL) {
                // one address pair: the immediate offset moves both sides
                indices_to_lds(pw + lane, lw, std::make_integer_sequence<int, kR8Chunks>{});
            } else {
#pragma unroll
                for (int j = 0; j < kR8Chunks; ++j)
                    if (in_range(j))
                        __builtin_amdgcn_global_load_lds((const void*)(pw + j * kWave + lane),
                                                         lw + j * kWave, 4, 0, 0);
            }
        }
        // All key loads, then the encoding: applied inside a per-key branch
        // it would make each load wait for the one before.  (Lanes past the
        // end get a code of 0; they are masked out everywhere below.)
        uint32_t key[kR8Chunks];
#pragma unroll
        for (int j = 0; j < kR8Chunks; ++j)
            key[j] = in_range(j) ? (uint32_t)__builtin_nontemporal_load(&kw[j * kWave + lane]) : 0u;
        if (code.pos | code.neg) {  // only the first pass of signed or float keys
#pragma unroll
            for (int j = 0; j < kR8Chunks; ++j) key[j] = code.apply(key[j]);
        }
        __syncthreads();

        // Rank chunk by chunk.  The peer group's lowest lane adds the group
        // size to the wave's count of the digit (an LDS add that returns
        // nothing), then every lane reads that count back: LDS carries out a
        // wave's operations in issue order, so the read sees this chunk's
        // add and no later one, and the key's rank is the count before the
        // group plus its peers in lower lanes.  No chunk waits on another.
        uint32_t rank[kR8Chunks];
#pragma unroll
        for (int j = 0; j < kR8Chunks; ++j) {
            const uint32_t d = (key[j] >> shift) & 255u;
            const uint64_t peers = FULL ? peers8_all(d) : peers8(d, in_range(j));
            const uint32_t below = lanes_below(peers);
            const uint32_t size = (uint32_t)__builtin_popcountll(peers);
            if (in_range(j) && below == 0) atomicAdd(&s_wh[w][d], size);
            rank[j] = s_wh[w][d] - size + below;
        }
        // the index loads were issued first: long done, and no stores yet
        if (WITH_PERM && HAS_PERM_IN) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();

        // Digit d (thread d): the tile's first slot of the digit (exclusive
        // scan of the totals over the 256 digits), then each wave's first
        // slot, and the offset from a slot to the global position.
        uint32_t c[kR8Waves];
        uint32_t tot = 0, inc = 0;
        if (threadIdx.x < kR8Digits) {
#pragma unroll
            for (int k = 0; k < kR8Waves; ++k) {
                c[k] = s_wh[k][threadIdx.x];
                tot += c[k];
            }
            inc = wave_incl_scan(tot);
            if (lane == kWave - 1) s_part[w] = inc;
        }
        __syncthreads();
        if (threadIdx.x < kR8Digits) {
            uint32_t first = inc - tot;
            for (int k = 0; k < w; ++k) first += s_part[k];
            s_off[threadIdx.x] = gbase - first;
#pragma unroll
            for (int k = 0; k < kR8Waves; ++k) {
                s_wh[k][threadIdx.x] = first;
                first += c[k];
            }
        }
        __syncthreads();

        // Sort the tile by digit in LDS, then write it out with consecutive
        // threads (each digit's keys form one contiguous output run).
#pragma unroll
        for (int j = 0; j < kR8Chunks; ++j) {
            rank[j] += s_wh[w][(key[j] >> shift) & 255u];  // now the slot
            if (FULL || (in_range(j) && rank[j] < kR8Tile)) s_stage[rank[j]] = key[j];
        }
        __syncthreads();
        // All staged keys, then their positions, then the stores: every LDS
        // read of the write-out in flight at once.  A position is clamped to
        // the row (it is inside always; the clamp keeps a corrupted offsets
        // table from writing out of bounds).
        const uint32_t last = (uint32_t)(len - 1);  // len <= INT32_MAX
        uint32_t sk[kR8Chunks], pos[kR8Chunks];
#pragma unroll
        for (int j = 0; j < kR8Chunks; ++j) sk[j] = s_stage[threadIdx.x + j * kR8Waves * kWave];
#pragma unroll
        for (int j = 0; j < kR8Chunks; ++j) {
            const uint32_t t = (uint32_t)threadIdx.x + j * kR8Waves * kWave;
            pos[j] = min(s_off[(sk[j] >> shift) & 255u] + t, last);
        }
        if (decode.pre | decode.one | decode.zero) {  // only the last pass of signed or float keys
#pragma unroll
            for (int j = 0; j < kR8Chunks; ++j) sk[j] = decode.apply(sk[j]);
        }
#pragma unroll
        for (int j = 0; j < kR8Chunks; ++j)
            if (FULL || threadIdx.x + j * kR8Waves * kWave < valid) kout[pos[j]] = (K)sk[j];
        if (WITH_PERM) {
            __syncthreads();
#pragma unroll
            for (int j = 0; j < kR8Chunks; ++j) {
                const int32_t pv = HAS_PERM_IN ? s_pin[(w * kR8Chunks + j) * kWave + lane]
                                               : (int32_t)(wbase + j * kWave + lane);
                if (FULL || (in_range(j) && rank[j] < kR8Tile)) s_stage[rank[j]] = (uint32_t)pv;
            }
            __syncthreads();
            int32_t* pout = perm_out + rbase;
#pragma unroll
            for (int j = 0; j < kR8Chunks; ++j) sk[j] = s_stage[threadIdx.x + j * kR8Waves * kWave];
#pragma unroll
            for (int j = 0; j < kR8Chunks; ++j)
                if (FULL || threadIdx.x + j * kR8Waves * kWave < valid) pout[pos[j]] = (int32_t)sk[j];
        }
    };
    if (full)
        body(std::true_type{});
    else
        body(std::false_type{});
}

// ---------------------------------------------------------------- driver

hipError_t launch_radix1_pass(const uint32_t* keys, const int32_t* idx_in, int bit,
                              uint32_t* keys_out, int32_t* idx_out, int64_t n, const uint64_t* hist,
                              void* ws, size_t ws_bytes, size_t status_offset, hipStream_t stream);

// 1-bit: header | final histogram | one status word per split tile |
//        per-block histograms.
// 4- and 8-bit: header | the count-table scan's workspace body | count table
//        (digits x tiles 32-bit counts, 16-byte aligned).
static int64_t radix1_status_words(int64_t n) { return (n + kR1Tile - 1) / kR1Tile; }
static int64_t r4_table_entries(int64_t n) { return r4_tiles(n) * 16; }
static size_t r4_table_offset(int64_t n) {
    return (scan1d_ws_bytes(r4_table_entries(n)) + 15) / 16 * 16;
}

size_t radix_ws_bytes(int64_t n, int bits) {
    if (bits == 8) return radix_rows_ws_bytes(1, n);
    if (bits == 4)
        return r4_table_offset(n) + (size_t)r4_table_entries(n) * sizeof(uint32_t);
    return kRadixStatusOffset + (size_t)radix1_status_words(n) * sizeof(uint64_t) +
           (size_t)kHistBlocks * kHistWords * sizeof(uint32_t);
}

constexpr KeyCode kIdentityCode{0u, 0u, 31};
constexpr KeyDecode kIdentityDecode{0u, 0u, 0u, 31};

// Rows of `len` keys (rows = 1: a 1-D sort of n = len keys), each sorted on
// its own by `passes` 8-bit passes over keys of type K (4 for 32-bit keys, 2
// for 16-bit), ping-ponging keys_tmp / keys_out (an even number of passes ends
// in keys_out); the first pass encodes the keys, the last one decodes them.
// Workspace: header | the table scan's workspace body | the count table.
static uint32_t r8_tpr(int64_t len) { return (uint32_t)((len + kR8Tile - 1) / kR8Tile); }
static size_t radix8_table_offset(int64_t rows, int64_t len) {
    const int64_t entries = (int64_t)kR8Digits * r8_tpr(len);
    const size_t scan = rows == 1 ? scan1d_ws_bytes(entries) : scan_rows_ws_bytes(rows, entries);
    return (scan + 15) / 16 * 16;
}
// rows x len keys within kMaxRadixKeys and a tile grid that fits one launch
// (the count table's row scan then fits its limits too).
bool radix_rows_fit(int64_t rows, int64_t len) {
    if (rows < 0 || len < 0) return false;
    if (rows == 0 || len == 0) return true;
    if (len > kMaxRadixKeys / rows) return false;
    return rows * (int64_t)r8_tpr(len) <= kMaxGridTiles;
}
size_t radix_rows_ws_bytes(int64_t rows, int64_t len) {
    return radix8_table_offset(rows, len) +
           (size_t)rows * kR8Digits * r8_tpr(len) * sizeof(uint32_t);
}

template <class K>
static hipError_t radix8_sort(const K* keys, K* keys_out, const int32_t* perm_in,
                              int32_t* perm_out, K* keys_tmp,
                              int32_t* perm_tmp, int64_t rows, int64_t len, int passes,
                              KeyCode code, KeyDecode decode, void* ws, hipStream_t stream) {
    const uint32_t tpr = r8_tpr(len);
    const uint32_t nt = (uint32_t)(rows * tpr);
    const int64_t entries = (int64_t)kR8Digits * tpr;  // per row
    const size_t toff = radix8_table_offset(rows, len);
    uint32_t* counts = reinterpret_cast<uint32_t*>(reinterpret_cast<char*>(ws) + toff);
    const K* src_k = keys;
    const int32_t* src_p = perm_out ? perm_in : nullptr;
    for (int p = 0; p < passes; ++p) {
        K* dk = (p % 2 == 0) ? keys_tmp : keys_out;
        int32_t* dp = perm_out ? ((p % 2 == 0) ? perm_tmp : perm_out) : nullptr;
        const KeyCode c = p == 0 ? code : kIdentityCode;
        const KeyDecode d = p == passes - 1 ? decode : kIdentityDecode;
        // 16-byte loads need every row start 16-byte aligned
        const bool vec = ((uintptr_t)src_k % 16) == 0 &&
                         (rows == 1 || ((size_t)len * sizeof(K)) % 16 == 0);
        hipLaunchKernelGGL(k_radix8_count<K>, dim3(nt), dim3(kR8Waves * kWave), 0, stream, src_k,
                           len, tpr, 8 * p, vec, counts, c);
        hipError_t e = rows == 1
                           ? launch_scan1d(Kind::I32, true, counts, counts, entries, nullptr,
                                           nullptr, ws, toff, stream)
                           : launch_scan_rows(Kind::I32, true, counts, counts, rows, entries, ws,
                                              toff, stream);
        if (e != hipSuccess) return e;
        auto k = dp ? (src_p ? k_radix8_scatter<K, true, true> : k_radix8_scatter<K, false, true>)
                    : k_radix8_scatter<K, false, false>;
        hipLaunchKernelGGL(k, dim3(nt), dim3(kR8Waves * kWave), 0, stream, src_k, src_p, dk, dp,
                           len, tpr, 8 * p, counts, c, d);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        src_k = dk;
        src_p = dp;
    }
    return hipSuccess;
}

hipError_t launch_radix_sort(const uint32_t* keys, uint32_t* keys_out, int32_t* perm_out,
                             uint32_t* keys_tmp, int32_t* perm_tmp, int64_t n, int bits, void* ws,
                             size_t ws_bytes, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    const int passes = 32 / bits;
    uint64_t* hist = reinterpret_cast<uint64_t*>(reinterpret_cast<char*>(ws) + kWsHeader);
    if (bits == 1) {
        uint32_t* part = reinterpret_cast<uint32_t*>(
            reinterpret_cast<char*>(ws) + kRadixStatusOffset + radix1_status_words(n) * sizeof(uint64_t));
        const int64_t hb64 = (n + 1023) / 1024;
        const int hb = (int)(hb64 < kHistBlocks ? hb64 : kHistBlocks);
        const bool vec = ((uintptr_t)keys % 16) == 0;
        hipLaunchKernelGGL(k_digit_hist, dim3(hb), dim3(256), 0, stream, keys, n, vec, part);
        hipLaunchKernelGGL(k_hist_reduce, dim3(1), dim3(1024), 0, stream, (const uint32_t*)part, hb, hist);
    }
    const uint32_t* src_k = keys;
    const int32_t* src_p = nullptr;
    for (int p = 0; p < passes; ++p) {
        uint32_t* dk = (p % 2 == 0) ? keys_tmp : keys_out;
        int32_t* dp = perm_out ? ((p % 2 == 0) ? perm_tmp : perm_out) : nullptr;
        if (bits == 1) {
            const hipError_t e = launch_radix1_pass(src_k, src_p, p, dk, dp, n, hist, ws, ws_bytes,
                                                    kRadixStatusOffset, stream);
            if (e != hipSuccess) return e;
        } else if (bits == 4) {
            const uint32_t nt = (uint32_t)r4_tiles(n);
            const size_t toff = r4_table_offset(n);
            uint32_t* counts = reinterpret_cast<uint32_t*>(reinterpret_cast<char*>(ws) + toff);
            const bool vec = ((uintptr_t)src_k % 16) == 0;
            hipLaunchKernelGGL(k_radix4_count, dim3(nt), dim3(kR4Waves * kWave), 0, stream, src_k, n,
                               4 * p, vec, counts, nt);
            hipError_t e = launch_scan1d(Kind::I32, true, counts, counts, r4_table_entries(n),
                                         nullptr, nullptr, ws, toff, stream);
            if (e != hipSuccess) return e;
            auto k = dp ? (src_p ? k_radix4_scatter<true, true> : k_radix4_scatter<false, true>)
                        : k_radix4_scatter<false, false>;
            hipLaunchKernelGGL(k, dim3(nt), dim3(kR4Waves * kWave), 0, stream, src_k, src_p, dk, dp,
                               n, 4 * p, counts, nt);
            e = hipGetLastError();
            if (e != hipSuccess) return e;
        } else {
            return radix8_sort<uint32_t>(keys, keys_out, nullptr, perm_out, keys_tmp, perm_tmp, 1,
                                         n, 4, kIdentityCode, kIdentityDecode, ws, stream);
        }
        src_k = dk;
        src_p = dp;
    }
    return hipSuccess;
}

hipError_t launch_radix_sort_typed(KeyType type, bool descending, const void* keys,
                                   void* keys_out, const int32_t* perm_in, int32_t* perm_out,
                                   void* keys_tmp,
                                   int32_t* perm_tmp, int64_t rows, int64_t len, void* ws,
                                   size_t ws_bytes, hipStream_t stream) {
    (void)ws_bytes;
    if (rows == 0 || len == 0) return hipSuccess;
    const bool wide = type != KeyType::F16;
    const uint32_t all = wide ? 0xFFFFFFFFu : 0xFFFFu;
    const uint32_t msb = wide ? 0x80000000u : 0x8000u;
    const int top = wide ? 31 : 15;
    KeyCode code{0u, 0u, top};
    KeyDecode decode{0u, 0u, 0u, top};
    switch (type) {
        case KeyType::U32:
            break;
        case KeyType::I32:  // two's complement: invert the sign bit
            code.pos = code.neg = msb;
            decode.one = decode.zero = msb;
            break;
        case KeyType::F32:
        case KeyType::F16:  // sign-magnitude: non-negative -> set the sign bit, negative -> invert all
            code.pos = msb;
            code.neg = all;
            decode.one = msb;   // code with the top bit set came from a non-negative key
            decode.zero = all;  // code with the top bit clear came from a negative key
            break;
    }
    if (descending) {
        code.pos ^= all;
        code.neg ^= all;
        decode.pre = all;
    }
    if (wide)
        return radix8_sort<uint32_t>((const uint32_t*)keys, (uint32_t*)keys_out, perm_in, perm_out,
                                     (uint32_t*)keys_tmp, perm_tmp, rows, len, 4, code, decode, ws,
                                     stream);
    return radix8_sort<uint16_t>((const uint16_t*)keys, (uint16_t*)keys_out, perm_in, perm_out,
                                 (uint16_t*)keys_tmp, perm_tmp, rows, len, 2, code, decode, ws,
                                 stream);
}

}  // namespace ls
