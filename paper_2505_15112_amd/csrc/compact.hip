// compact.hip -- scan-based data movement: Compress and Split (Section 5).
//
// Compress (torch.masked_select): keep x_i where mask_i != 0, in index order.
// The exclusive count of kept elements before i is their output position; it
// is a scan of 0/1 flags, computed tile-locally (lane serial + DPP wavefront
// + LDS) and carried between tiles by decoupled look-back on the counts --
// one kernel, one pass: mask and values read once, kept values written once.
//
// Split (SplitInd): stable two-way partition with source indices.  Flagged
// element i goes to e_i (exclusive count of flagged before it), unflagged to
// n_true + (i - e_i).  n_true must be known before any tile stores, so a
// small counting kernel runs first (reading only the flag bytes, each block
// storing its own partial count), and every split tile adds the partials.  As
// the pass of the one-bit radix sort (Section 5), the flag is "key bit b is
// 0" and n_true comes from the sort's digit histogram instead.
//
// Both kernels store through LDS: the elements of one wavefront chunk that go
// to one contiguous output run are gathered first, then written by
// consecutive lanes, so the stores are dense rather than scattered dwords.
#include <limits.h>

#include "launch.hpp"
#include "tile.hpp"

namespace ls {

static inline int64_t s_tiles(int64_t n);

// Per byte: 1 if the byte is non-zero, else 0 (bits 0, 8, 16, 24).
__device__ __forceinline__ uint32_t nonzero_bytes(uint32_t m) {
    uint32_t t = m | ((m >> 4) & 0x0f0f0f0fu);
    t |= (t >> 2) & 0x33333333u;
    t |= (t >> 1) & 0x55555555u;
    return t & 0x01010101u;
}

// The flag-counting kernel runs this many blocks; each writes its count to
// one 64-bit workspace word after the split's status words.
constexpr int kCountBlocks = 256;

// ---------------------------------------------------------------- compress

// Compress tile: 8 waves x 16 chunks x 64 lanes x 4 elements = 32768.  A
// lane keeps the 4 mask bytes of a chunk packed in one register (bit 8e set
// when element e is kept) next to its 4 values, so a large tile fits in
// registers and the per-tile look-back is paid rarely.
constexpr int kPWaves = 8;
constexpr int kPChunks = 16;
constexpr int kPStage = 4;  // chunks staged per write-out (with indices)
constexpr int64_t kPTile = kPWaves * kPChunks * kWave * 4;

template <bool VEC, bool WITH_IDX, int WAVES, int CHUNKS>
__global__ __launch_bounds__(WAVES* kWave) LS_OCCUPANCY4 void k_compact(
    const float* x, const uint8_t* mask, float* out, int32_t* idx, int32_t* count, int64_t n,
    WsHeader* hdr, uint64_t* status, int64_t status_words, uint32_t ntiles) {
    static_assert(WAVES * CHUNKS * kWave * 4 == kPTile, "one compaction tile size");
    __shared__ Ticket s_ticket;
    __shared__ uint32_t s_wtot[WAVES];
    __shared__ uint32_t s_carry;
    // STAGE chunks of kept values (and indices) per wave between stores: as
    // many as leave room in LDS for two workgroups per CU (values only on the
    // 8-wave tile: twice as many)
    constexpr int STAGE = WAVES > kPWaves ? kPStage / 2 : (WITH_IDX ? kPStage : 2 * kPStage);
    static_assert(CHUNKS % STAGE == 0, "whole batches of chunks");
    __shared__ __align__(16) float s_val[WAVES][kWave * 4 * STAGE + 4];
    __shared__ __align__(16) int32_t s_idx[WITH_IDX ? WAVES : 1][kWave * 4 * STAGE + 4];

    if (threadIdx.x == 0) s_ticket = take_ticket(hdr, ntiles);
    __syncthreads();
    const uint32_t tile32 = (uint32_t)__builtin_amdgcn_readfirstlane(s_ticket.tile);
    const uint32_t epoch = (uint32_t)__builtin_amdgcn_readfirstlane(s_ticket.epoch);
    if (tile32 >= ntiles) {
        if (threadIdx.x == 0)
            __hip_atomic_store(&hdr->error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return;
    }
    const int64_t tile = tile32;
    const int64_t base = tile * kPTile;
    const int lane = lane_id();
    const int w = threadIdx.x / kWave;
    auto offset = [&](int j) { return base + ((int64_t)(w * CHUNKS + j) * kWave + lane) * 4; };

    uint32_t kept[CHUNKS];
    float xv[CHUNKS][4];
    if (VEC && base + kPTile <= n) {
        // All mask loads first: the tile's count (and so its look-back) needs
        // only them, and the value loads stay in flight meanwhile.
#pragma unroll
        for (int j = 0; j < CHUNKS; ++j)
            kept[j] = nonzero_bytes(*reinterpret_cast<const uint32_t*>(mask + offset(j)));
#pragma unroll
        for (int j = 0; j < CHUNKS; ++j) load_vec<float, float, 4, true>(x + offset(j), xv[j]);
    } else {
#pragma unroll
        for (int j = 0; j < CHUNKS; ++j) {
            const int64_t off = offset(j);
            kept[j] = 0;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                xv[j][e] = 0.f;
                if (off + e < n) {
                    kept[j] |= (uint32_t)(mask[off + e] != 0) << (8 * e);
                    xv[j][e] = x[off + e];
                }
            }
        }
    }
    // lane counts -> wavefront scans -> tile total
    uint32_t lane_off[CHUNKS];
    uint32_t run = 0;
#pragma unroll
    for (int j = 0; j < CHUNKS; ++j) {
        const uint32_t c = (uint32_t)__builtin_popcount(kept[j]);
        const uint32_t inc = wave_incl_scan(c);
        lane_off[j] = run + inc - c;
        run += lane_read(inc, kWave - 1);
    }
    if (lane == 0) s_wtot[w] = run;
    __syncthreads();
    uint32_t wofs = 0, agg = 0;
#pragma unroll
    for (int k = 0; k < WAVES; ++k) {
        const uint32_t t = s_wtot[k];
        if (k < w) wofs += t;
        agg += t;
    }
    if (threadIdx.x < kWave) {
        const uint32_t excl = lookback<uint32_t>(status, tile32, 0u, agg, 0u, epoch, hdr);
        if (threadIdx.x == 0) {
            s_carry = excl;
            if (tile == ntiles - 1) *count = (int32_t)(excl + agg);
            finish_epoch(hdr, epoch, ntiles, status, status_words);
        }
    }
    __syncthreads();
    // The kept elements of a batch of STAGE consecutive chunks form one
    // contiguous output run: gather them in this wave's LDS slot, then write
    // the run with consecutive lanes (one LDS round trip per batch).
    const uint32_t c0 = s_carry + wofs;
    float* st = s_val[w];
    int32_t* si = s_idx[WITH_IDX ? w : 0];
    // Values only: 16-byte stores of the runs' interiors when the output
    // allows them (the run is staged at its destination's index mod 4, so
    // that LDS and memory quads line up; a uniform choice).  Measured 375 ->
    // 369 us at n = 2^28; with indices as well no gain, so that kernel keeps
    // the 4-byte stores.
    const bool quads = VEC && !WITH_IDX && ((uintptr_t)out & 15) == 0;
#pragma unroll
    for (int j0 = 0; j0 < CHUNKS; j0 += STAGE) {
        const uint32_t run0 = lane_read(lane_off[j0], 0);  // kept before this batch, in the wave
        const uint32_t dst = c0 + run0;
        const uint32_t sh = quads ? (dst & 3u) : 0u;
#pragma unroll
        for (int j = j0; j < j0 + STAGE; ++j) {
            const int64_t off = offset(j);
            uint32_t r = sh + lane_off[j] - run0;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                if ((kept[j] >> (8 * e)) & 1u) {
                    st[r] = xv[j][e];
                    if (WITH_IDX) si[r] = (int32_t)(off + e);
                    ++r;
                }
            }
        }
        const uint32_t cnt =
            (j0 + STAGE < CHUNKS ? lane_read(lane_off[j0 + STAGE], 0) : run) - run0;
        wave_lds_sync();
        if (quads) {
            // quads of [dst - sh, dst + cnt): slots s .. s + 3 of the stage hold
            // output elements dst - sh + s ..; slots below sh or at sh + cnt and
            // above are not this run's
            const uint32_t a0 = dst - sh;
            const uint32_t nq = (sh + cnt + 3u) / 4u;
            for (uint32_t q = lane; q < nq; q += kWave) {
                const uint32_t s0 = 4u * q;
                if (s0 >= sh && s0 + 4u <= sh + cnt && (uint64_t)a0 + s0 + 4u <= (uint64_t)n) {
                    *reinterpret_cast<float4*>(out + a0 + s0) = *reinterpret_cast<const float4*>(st + s0);
                    if (WITH_IDX)
                        *reinterpret_cast<int4*>(idx + a0 + s0) = *reinterpret_cast<const int4*>(si + s0);
                } else {
#pragma unroll
                    for (uint32_t e = 0; e < 4; ++e) {
                        const uint32_t sl = s0 + e;
                        if (sl >= sh && sl < sh + cnt && (uint64_t)a0 + sl < (uint64_t)n) {
                            out[a0 + sl] = st[sl];
                            if (WITH_IDX) idx[a0 + sl] = si[sl];
                        }
                    }
                }
            }
        } else {
            for (uint32_t t = lane; t < cnt; t += kWave) {
                if (dst + t < (uint64_t)n) {  // always true; guards the write against a bad count
                    out[dst + t] = st[t];
                    if (WITH_IDX) idx[dst + t] = si[t];
                }
            }
        }
        wave_lds_sync();
    }
}

// ---------------------------------------------------------------- split

// Count the non-zero flag bytes: kCountBlocks blocks of 1024 threads,
// grid-stride, 16 flags per 16-byte load, 4 loads in flight per thread; every
// block stores its count in part[blockIdx.x] (no atomics: the split kernel
// sums the partials).
__global__ __launch_bounds__(1024) void k_count_flags(const uint8_t* flags, int64_t n, bool vec,
                                                      uint64_t* part) {
    __shared__ uint32_t s_part[16];
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t t0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    uint32_t cnt = 0;
    int64_t done = 0;
    if (vec) {
        const u32x4* f4 = reinterpret_cast<const u32x4*>(flags);
        const int64_t n16 = n / 16;
        for (int64_t i = t0; i < n16; i += 4 * stride) {
            u32x4 v[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int64_t q = i + u * stride;
                v[u] = q < n16 ? f4[q] : u32x4{0, 0, 0, 0};
            }
#pragma unroll
            for (int u = 0; u < 4; ++u)
                cnt += __builtin_popcount(nonzero_bytes(v[u].x)) + __builtin_popcount(nonzero_bytes(v[u].y)) +
                       __builtin_popcount(nonzero_bytes(v[u].z)) + __builtin_popcount(nonzero_bytes(v[u].w));
        }
        done = n16 * 16;
    }
    for (int64_t i = done + t0; i < n; i += stride) cnt += flags[i] != 0;
    const uint32_t wsum = wave_sum(cnt);
    if (lane_id() == 0) s_part[threadIdx.x / kWave] = wsum;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t t = 0;
        for (int k = 0; k < 16; ++k) t += s_part[k];
        part[blockIdx.x] = t;
    }
}

// Sum of the kCountBlocks partial counts, by one full wavefront.
__device__ __forceinline__ uint32_t sum_partials(const uint64_t* part) {
    uint32_t v = 0;
    for (int i = lane_id(); i < kCountBlocks; i += kWave) v += (uint32_t)part[i];
    return wave_sum(v);
}

// Number of keys whose bit `bit` is 0, from the 8 x 16 digit histogram of
// the radix sort (digit position bit / 4).
__device__ __forceinline__ uint32_t zeros_of_bit(const uint64_t* hist, int bit) {
    uint32_t z = 0;
    for (int v = 0; v < 16; ++v)
        if (((v >> (bit & 3)) & 1) == 0) z += (uint32_t)hist[(bit >> 2) * 16 + v];
    return z;
}

// Split tile: 8 waves x 8 chunks x 64 lanes x 4 elements = 16384.  Flags are
// kept packed (bit 8e of one register per chunk), keys and source indices in
// registers.  hist == nullptr: n_true comes from the counting kernel's header
// word; otherwise (radix-sort pass) it is derived from the digit histogram.
constexpr int kSWaves = 8;
constexpr int kSChunks = 8;
constexpr int64_t kSTile = kSWaves * kSChunks * kWave * 4;

template <bool FROM_BITS, bool VEC, bool HAS_IDX_IN, bool WITH_IDX, int CHUNKS>
__global__ __launch_bounds__(kSWaves* kWave) LS_OCCUPANCY4 void k_split(
    const uint32_t* keys, const int32_t* idx_in, const uint8_t* flags, int bit, uint32_t* keys_out,
    int32_t* idx_out, int32_t* n_true_out, int64_t n, WsHeader* hdr, uint64_t* status,
    int64_t status_words, uint32_t ntiles, const uint64_t* hist, const uint64_t* part) {
    __shared__ Ticket s_ticket;
    __shared__ uint32_t s_wtot[kSWaves];
    __shared__ uint32_t s_carry;
    __shared__ uint32_t s_ntrue;
    __shared__ uint32_t s_key[kSWaves][kWave * 4];
    __shared__ int32_t s_idx[WITH_IDX ? kSWaves : 1][kWave * 4];

    if (threadIdx.x == 0) s_ticket = take_ticket(hdr, ntiles);
    __syncthreads();
    const uint32_t tile32 = (uint32_t)__builtin_amdgcn_readfirstlane(s_ticket.tile);
    const uint32_t epoch = (uint32_t)__builtin_amdgcn_readfirstlane(s_ticket.epoch);
    if (tile32 >= ntiles) {
        if (threadIdx.x == 0)
            __hip_atomic_store(&hdr->error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return;
    }
    const int64_t tile = tile32;
    constexpr int64_t kTile = (int64_t)kSWaves * CHUNKS * kWave * 4;
    const int64_t base = tile * kTile;
    const int lane = lane_id();
    const int w = threadIdx.x / kWave;
    auto offset = [&](int j) { return base + ((int64_t)(w * CHUNKS + j) * kWave + lane) * 4; };
    if (threadIdx.x < kWave) {
        const uint32_t nt = hist ? zeros_of_bit(hist, bit) : sum_partials(part);
        if (threadIdx.x == 0) s_ntrue = nt;
    }

    uint32_t k[CHUNKS][4];
    int32_t iv[CHUNKS][4];
    uint32_t fl[CHUNKS];  // bit 8e: element e is flagged
    const bool full = base + kTile <= n;
    if (VEC && full) {
        // Loads in the order the tile's count needs them (flags, or the keys
        // whose bit is the flag), source indices last.
        if (!FROM_BITS) {
#pragma unroll
            for (int j = 0; j < CHUNKS; ++j)
                fl[j] = nonzero_bytes(*reinterpret_cast<const uint32_t*>(flags + offset(j)));
        }
#pragma unroll
        for (int j = 0; j < CHUNKS; ++j) load_vec<uint32_t, uint32_t, 4, true>(keys + offset(j), k[j]);
        if (HAS_IDX_IN) {
#pragma unroll
            for (int j = 0; j < CHUNKS; ++j) load_vec<int32_t, int32_t, 4, true>(idx_in + offset(j), iv[j]);
        }
    } else {
#pragma unroll
        for (int j = 0; j < CHUNKS; ++j) {
            const int64_t off = offset(j);
            fl[j] = 0;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const bool ok = off + e < n;
                k[j][e] = ok ? keys[off + e] : 0u;
                if (HAS_IDX_IN) iv[j][e] = ok ? idx_in[off + e] : 0;
                if (!FROM_BITS && ok) fl[j] |= (uint32_t)(flags[off + e] != 0) << (8 * e);
            }
        }
    }
    if (FROM_BITS) {
#pragma unroll
        for (int j = 0; j < CHUNKS; ++j) {
            const int64_t off = offset(j);
            fl[j] = 0;
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (full || off + e < n) fl[j] |= (((k[j][e] >> bit) & 1u) ^ 1u) << (8 * e);
        }
    }
    uint32_t lane_off[CHUNKS];
    uint32_t run = 0;
#pragma unroll
    for (int j = 0; j < CHUNKS; ++j) {
        const uint32_t c = (uint32_t)__builtin_popcount(fl[j]);  // (split: s_ntrue set before the barrier below)
        const uint32_t inc = wave_incl_scan(c);
        lane_off[j] = run + inc - c;
        run += lane_read(inc, kWave - 1);
    }
    if (lane == 0) s_wtot[w] = run;
    __syncthreads();
    uint32_t wofs = 0, agg = 0;
#pragma unroll
    for (int q = 0; q < kSWaves; ++q) {
        const uint32_t t = s_wtot[q];
        if (q < w) wofs += t;
        agg += t;
    }
    if (threadIdx.x < kWave) {
        const uint32_t excl = lookback<uint32_t>(status, tile32, 0u, agg, 0u, epoch, hdr);
        if (threadIdx.x == 0) {
            s_carry = excl;
            if (tile == 0 && n_true_out) *n_true_out = (int32_t)s_ntrue;
            finish_epoch(hdr, epoch, ntiles, status, status_words);
        }
    }
    __syncthreads();
    // A chunk's flagged keys form one contiguous output run and its other
    // keys another: gather both in this wave's LDS slot (flagged first), then
    // write the two runs with consecutive lanes.
    const uint32_t c0 = s_carry + wofs;
    const uint32_t n_true = s_ntrue;
    uint32_t* sk = s_key[w];
    int32_t* si = s_idx[WITH_IDX ? w : 0];
#pragma unroll
    for (int j = 0; j < CHUNKS; ++j) {
        const int64_t off = offset(j);
        const int64_t g0 = base + (int64_t)(w * CHUNKS + j) * kWave * 4;  // chunk start
        const uint32_t run0 = lane_read(lane_off[j], 0);
        const uint32_t cnt = (j + 1 < CHUNKS ? lane_read(lane_off[j + 1], 0) : run) - run0;
        const int64_t valid64 = n - g0 < kWave * 4 ? n - g0 : kWave * 4;
        const uint32_t valid = valid64 > 0 ? (uint32_t)valid64 : 0u;
        uint32_t r = lane_off[j] - run0;  // flagged before this element, in the chunk
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const uint32_t le = (uint32_t)lane * 4 + e;  // element index in the chunk
            if (le < valid) {
                const bool flagged = (fl[j] >> (8 * e)) & 1u;
                const uint32_t slot = flagged ? r : cnt + (le - r);
                sk[slot] = k[j][e];
                if (WITH_IDX) si[slot] = HAS_IDX_IN ? iv[j][e] : (int32_t)(off + e);
                r += flagged;
            }
        }
        wave_lds_sync();
        const uint32_t true_dst = c0 + run0;                        // flagged before the chunk
        const uint32_t false_dst = n_true + (uint32_t)g0 - true_dst;  // unflagged before it
        for (uint32_t t = lane; t < valid; t += kWave) {
            const uint32_t pos = t < cnt ? true_dst + t : false_dst + (t - cnt);
            if (pos < (uint64_t)n) {  // always true; guards the write against a bad count
                keys_out[pos] = sk[t];
                if (WITH_IDX) idx_out[pos] = si[t];
            }
        }
        wave_lds_sync();
    }
}

static inline int64_t s_tiles(int64_t n) { return (n + kSTile - 1) / kSTile; }

// ---------------------------------------------------------------- launchers

// Sized for the split tile (the smaller one; compress uses fewer words), then
// the flag counter's per-block partials.
static size_t split_part_offset(int64_t n) { return kWsHeader + (size_t)s_tiles(n) * sizeof(uint64_t); }
size_t compact_ws_bytes(int64_t n) { return split_part_offset(n) + kCountBlocks * sizeof(uint64_t); }

static bool al(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

__global__ void k_zero_count(int32_t* count) {
    if (threadIdx.x == 0) *count = 0;
}

hipError_t launch_compact(const float* x, const uint8_t* mask, float* out, int32_t* idx,
                          int32_t* count, int64_t n, void* ws, size_t ws_bytes,
                          hipStream_t stream) {
    if (n == 0) {
        hipLaunchKernelGGL(k_zero_count, dim3(1), dim3(64), 0, stream, count);
        return hipGetLastError();
    }
    const uint32_t nt = (uint32_t)((n + kPTile - 1) / kPTile);
    WsHeader* hdr = reinterpret_cast<WsHeader*>(ws);
    uint64_t* status = reinterpret_cast<uint64_t*>(reinterpret_cast<char*>(ws) + kWsHeader);
    const int64_t sw = (int64_t)((ws_bytes - kWsHeader) / sizeof(uint64_t));
    const bool vec = al(x, 16) && al(mask, 4);
    // Misaligned data is loaded element by element, which needs more
    // registers per element: the same tile as 16 waves x 8 chunks.
    auto k = vec ? (idx ? k_compact<true, true, kPWaves, kPChunks> : k_compact<true, false, kPWaves, kPChunks>)
                 : (idx ? k_compact<false, true, 2 * kPWaves, kPChunks / 2>
                        : k_compact<false, false, 2 * kPWaves, kPChunks / 2>);
    const unsigned threads = (vec ? kPWaves : 2 * kPWaves) * kWave;
    hipLaunchKernelGGL(k, dim3(nt), dim3(threads), 0, stream, x, mask, out, idx, count, n, hdr,
                       status, sw, nt);
    return hipGetLastError();
}

// Tiles of kSWaves x CHUNKS x 64 x 4 elements.  With aligned data, flags from
// a mask and no input indices a lane holds 4 keys and a packed flag word per
// chunk, so 16 chunks fit the register budget (32768-element tiles); the
// other forms need more registers per element and take 8 (16384).
template <bool FROM_BITS, bool VEC, bool HAS_IDX_IN>
static void split_launch(const uint32_t* keys, const int32_t* idx_in, const uint8_t* flags, int bit,
                         uint32_t* keys_out, int32_t* idx_out, int32_t* n_true_out, int64_t n,
                         WsHeader* hdr, uint64_t* status, int64_t sw, const uint64_t* hist,
                         const uint64_t* part, hipStream_t stream) {
    constexpr int CHUNKS = (VEC && !HAS_IDX_IN && !FROM_BITS) ? 2 * kSChunks : kSChunks;
    constexpr int64_t tile = (int64_t)kSWaves * CHUNKS * kWave * 4;
    const uint32_t nt = (uint32_t)((n + tile - 1) / tile);
    auto k = idx_out ? k_split<FROM_BITS, VEC, HAS_IDX_IN, true, CHUNKS>
                     : k_split<FROM_BITS, VEC, HAS_IDX_IN, false, CHUNKS>;
    hipLaunchKernelGGL(k, dim3(nt), dim3(kSWaves * kWave), 0, stream, keys, idx_in, flags, bit,
                       keys_out, idx_out, n_true_out, n, hdr, status, sw, nt, hist, part);
}

template <bool FROM_BITS, bool VEC>
static void split_launch_any(const uint32_t* keys, const int32_t* idx_in, const uint8_t* flags,
                             int bit, uint32_t* keys_out, int32_t* idx_out, int32_t* n_true_out,
                             int64_t n, WsHeader* hdr, uint64_t* status, int64_t sw,
                             const uint64_t* hist, const uint64_t* part, hipStream_t stream) {
    if (idx_in)
        split_launch<FROM_BITS, VEC, true>(keys, idx_in, flags, bit, keys_out, idx_out, n_true_out,
                                           n, hdr, status, sw, hist, part, stream);
    else
        split_launch<FROM_BITS, VEC, false>(keys, idx_in, flags, bit, keys_out, idx_out, n_true_out,
                                            n, hdr, status, sw, hist, part, stream);
}

// One LSB radix-sort pass on key bit `bit` (flag = bit is 0), with the count
// of zero bits taken from the digit histogram `hist`.
hipError_t launch_radix1_pass(const uint32_t* keys, const int32_t* idx_in, int bit,
                              uint32_t* keys_out, int32_t* idx_out, int64_t n, const uint64_t* hist,
                              void* ws, size_t ws_bytes, size_t status_offset, hipStream_t stream) {
    WsHeader* hdr = reinterpret_cast<WsHeader*>(ws);
    uint64_t* status = reinterpret_cast<uint64_t*>(reinterpret_cast<char*>(ws) + status_offset);
    const int64_t sw = (int64_t)((ws_bytes - status_offset) / sizeof(uint64_t));
    const bool vec = al(keys, 16) && (!idx_in || al(idx_in, 16));
    if (vec)
        split_launch_any<true, true>(keys, idx_in, nullptr, bit, keys_out, idx_out, nullptr, n, hdr,
                                     status, sw, hist, nullptr, stream);
    else
        split_launch_any<true, false>(keys, idx_in, nullptr, bit, keys_out, idx_out, nullptr, n,
                                      hdr, status, sw, hist, nullptr, stream);
    return hipGetLastError();
}

hipError_t launch_split(const uint32_t* keys, const int32_t* idx_in, const uint8_t* flags, int bit,
                        uint32_t* keys_out, int32_t* idx_out, int32_t* n_true_out, int64_t n,
                        void* ws, size_t ws_bytes, hipStream_t stream) {
    (void)bit;
    if (n == 0) {
        if (n_true_out) hipLaunchKernelGGL(k_zero_count, dim3(1), dim3(64), 0, stream, n_true_out);
        return hipGetLastError();
    }
    WsHeader* hdr = reinterpret_cast<WsHeader*>(ws);
    uint64_t* status = reinterpret_cast<uint64_t*>(reinterpret_cast<char*>(ws) + kWsHeader);
    // (the epoch-wrap clear may zero the partial counts too: they are read
    // before any workgroup finishes)
    const int64_t sw = (int64_t)((ws_bytes - kWsHeader) / sizeof(uint64_t));
    uint64_t* part = reinterpret_cast<uint64_t*>(reinterpret_cast<char*>(ws) + split_part_offset(n));
    hipLaunchKernelGGL(k_count_flags, dim3(kCountBlocks), dim3(1024), 0, stream, flags, n,
                       ((uintptr_t)flags % 16) == 0, part);
    const bool vec = al(keys, 16) && (!idx_in || al(idx_in, 16)) && al(flags, 4);
    if (vec)
        split_launch_any<false, true>(keys, idx_in, flags, 0, keys_out, idx_out, n_true_out, n, hdr,
                                      status, sw, nullptr, part, stream);
    else
        split_launch_any<false, false>(keys, idx_in, flags, 0, keys_out, idx_out, n_true_out, n,
                                       hdr, status, sw, nullptr, part, stream);
    return hipGetLastError();
}

}  // namespace ls
