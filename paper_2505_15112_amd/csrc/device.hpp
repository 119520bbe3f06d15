// device.hpp -- wavefront and cross-workgroup primitives for gfx950 (CDNA4).
//
//  * wave64 inclusive / exclusive add-scan by DPP (row_shr 1,2,4,8 inside each
//    16-lane row, then row_bcast:15 and row_bcast:31 across rows);
//  * packed 64-bit tile status words (state in bits 63..62, 32-bit payload in
//    bits 31..0) read and written with relaxed agent-scope atomics, so that a
//    state and its value are always observed together without fences;
//  * the decoupled look-back of Merrill and Garland (cited in Section 2.1 of
//    the paper): a tile publishes its aggregate, then one wavefront walks back
//    over 64 predecessors per load, adding aggregates until it meets an
//    inclusive prefix, and finally publishes its own inclusive prefix.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

// Register budget of the tile kernels: at least 4 waves per SIMD, i.e. at
// most 128 VGPRs, so 16 waves share a CU (two 8-wave workgroups, four 4-wave
// ones or one of 16).  A tile's data lives in registers from its loads to its
// stores, so this is what bounds the bytes in flight per CU.
#define LS_OCCUPANCY4 __attribute__((amdgpu_waves_per_eu(4)))
// At most 64 VGPRs (8 waves per SIMD): for short tile kernels launched with
// about as many workgroups as fit the chip at that occupancy, so that none
// waits for a free slot.
#define LS_OCCUPANCY8 __attribute__((amdgpu_waves_per_eu(8)))

namespace ls {

constexpr int kWave = 64;

// ---------------------------------------------------------------- scalar ops

template <class T>
struct Bits;
template <>
struct Bits<uint32_t> {
    __device__ static uint32_t to(uint32_t v) { return v; }
    __device__ static uint32_t from(uint32_t b) { return b; }
};
template <>
struct Bits<float> {
    __device__ static uint32_t to(float v) { return __builtin_bit_cast(uint32_t, v); }
    __device__ static float from(uint32_t b) { return __builtin_bit_cast(float, b); }
};

// DPP move with zero for lanes whose source is outside the row / disabled.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint32_t dpp0(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, ROW_MASK, 0xf, false);
}

template <int CTRL, int ROW_MASK, class T>
__device__ __forceinline__ T dpp_add(T v) {
    return v + Bits<T>::from(dpp0<CTRL, ROW_MASK>(Bits<T>::to(v)));
}

// Inclusive add-scan over the 64 lanes of a wavefront.
template <class T>
__device__ __forceinline__ T wave_incl_scan(T v) {
    v = dpp_add<0x111, 0xf>(v);  // row_shr:1
    v = dpp_add<0x112, 0xf>(v);  // row_shr:2
    v = dpp_add<0x114, 0xf>(v);  // row_shr:4
    v = dpp_add<0x118, 0xf>(v);  // row_shr:8   -> prefix inside each 16-lane row
    v = dpp_add<0x142, 0xa>(v);  // row_bcast:15 into rows 1 and 3
    v = dpp_add<0x143, 0xc>(v);  // row_bcast:31 into rows 2 and 3
    return v;
}

// Exclusive scan from the inclusive one: shift the whole wave right by a lane.
template <class T>
__device__ __forceinline__ T wave_shr1(T incl) {
    return Bits<T>::from(dpp0<0x138, 0xf>(Bits<T>::to(incl)));  // wave_shr:1, lane 0 gets 0
}

template <class T>
__device__ __forceinline__ T lane_read(T v, int lane) {
    return Bits<T>::from((uint32_t)__builtin_amdgcn_readlane((int)Bits<T>::to(v), lane));
}

// Sum over the wave, returned to every lane (wave-uniform).
template <class T>
__device__ __forceinline__ T wave_sum(T v) {
    return lane_read(wave_incl_scan(v), kWave - 1);
}

__device__ __forceinline__ int lane_id() { return (int)__lane_id(); }

// Orders one wavefront's LDS writes before its later LDS reads of other
// lanes' data (the LDS executes a wave's instructions in order; this keeps
// the compiler from moving the accesses across).
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// ---------------------------------------------------------------- test pauses

// Test builds (LS_ADVERSARIAL_DELAYS defined) pause for a pseudo-random time
// before each step of the inter-workgroup protocols -- after taking a tile
// ticket, before publishing a status word, before arriving at a row counter
// -- so that workgroups reach those steps in orders a normal run seldom
// produces: usually 0-3 us, one time in eight 14-30 us.  Product builds
// compile it away.  Called by one thread or one wavefront at a time.
#ifdef LS_ADVERSARIAL_DELAYS
__device__ __forceinline__ void adversarial_pause(uint32_t key) {
    uint32_t h = key * 0x9E3779B1u ^ (uint32_t)__builtin_amdgcn_s_memrealtime();
    h ^= h >> 15;
    h *= 0x2C1B3C6Du;
    h ^= h >> 12;
    const uint32_t rounds = (h & 7u) == 0 ? 64u + ((h >> 3) & 63u) : (h >> 3) & 15u;
    for (uint32_t i = 0; i < rounds; ++i) __builtin_amdgcn_s_sleep(8);  // 512 cycles
}
#else
__device__ __forceinline__ void adversarial_pause(uint32_t) {}
#endif

// ---------------------------------------------------------------- workspace

// Every workspace starts with a 256-byte header:
//   [0, 8)    ticket word: bits 63..32 epoch, bits 31..0 next tile ticket
//   [8, 12)   done counter, used only by the call that wraps the epoch
//   [12, 16)  error flag: set to 1 if a look-back gave up waiting (the
//             workspace was not zero-filled before first use)
//   [16, 256) reserved
// A zero-filled workspace is ready; after that every look-back kernel leaves
// it ready for the next call: the workgroup that takes the last ticket resets
// the ticket count and advances the epoch, and status words are tagged with
// the epoch of the call that wrote them, so words left by earlier calls read
// as "nothing published yet".  No per-call clearing is needed.
// Invariant kept by every op: outside the header, every 64-bit workspace word
// either has its two top bits 0 (state "nothing published": zero, or scratch
// such as per-block partial counts and sums, which are always below 2^30) or
// is a status word of an epoch no later than the current one.  So any
// workspace can serve any sequence of calls.
struct WsHeader {
    uint64_t ticket;
    uint32_t done;
    uint32_t error;
    uint64_t reserved[30];
};
static_assert(sizeof(WsHeader) == 256, "workspace header is 256 bytes");

struct Ticket {
    uint32_t tile;
    uint32_t epoch;
};

// Taken by one thread per workgroup.  Tickets are handed out in the order
// workgroups get here, so every tile a workgroup waits on belongs to a
// workgroup that is already running.
__device__ __forceinline__ Ticket take_ticket(WsHeader* h, uint32_t nwg) {
    const uint64_t old =
        __hip_atomic_fetch_add(&h->ticket, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    Ticket t{(uint32_t)old, (uint32_t)(old >> 32)};
    if (t.tile == nwg - 1)  // every other ticket of this launch is taken
        __hip_atomic_store(&h->ticket, (uint64_t)(t.epoch + 1) << 32, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
    adversarial_pause(t.tile);
    return t;
}

// ---------------------------------------------------------------- tile status

// Status word: bits 63..62 state, bits 61..32 epoch (low 30 bits), 31..0 value.
constexpr uint64_t kStateShift = 62;
constexpr uint64_t kStateMask = 3ull << kStateShift;
constexpr uint64_t kStateX = 0;                    // nothing published yet
constexpr uint64_t kStateA = 1ull << kStateShift;  // tile aggregate
constexpr uint64_t kStateP = 2ull << kStateShift;  // inclusive prefix
constexpr uint32_t kEpochMask = (1u << 30) - 1;
constexpr uint32_t kSpinLimit = 1u << 20;

__device__ __forceinline__ uint64_t status_word(uint64_t state, uint32_t epoch, uint32_t bits) {
    return state | ((uint64_t)(epoch & kEpochMask) << 32) | bits;
}
// State of a word as seen by a call of this epoch (stale words read as X).
__device__ __forceinline__ uint64_t status_state(uint64_t s, uint32_t epoch) {
    return ((uint32_t)(s >> 32) & kEpochMask) == (epoch & kEpochMask) ? (s & kStateMask) : kStateX;
}
__device__ __forceinline__ uint64_t status_load(uint64_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void status_store(uint64_t* p, uint64_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Decoupled look-back, run by ONE full wavefront of the tile's workgroup.
// Tiles [first, tile) precede `tile` in its scan segment; `first` publishes
// base + agg as its inclusive prefix directly.  Returns the exclusive prefix
// of `tile` (which includes base) to every lane and publishes the inclusive
// prefix of `tile`.  Spins (with s_sleep) only on predecessors that have not
// published yet; they hold earlier tickets, so they are running and the wait
// ends.  The spin is bounded all the same: after kSpinLimit rounds it raises
// the workspace error flag and carries on with a wrong value rather than hang.
template <class T, int K = 1>
__device__ T lookback(uint64_t* status, uint32_t tile, uint32_t first, T agg, T base,
                      uint32_t epoch, WsHeader* h) {
    const int lane = lane_id();
    if (lane == 0) adversarial_pause(tile);
    if (tile == first) {
        if (lane == 0) status_store(status + tile, status_word(kStateP, epoch, Bits<T>::to(base + agg)));
        return base;
    }
    if (lane == 0) status_store(status + tile, status_word(kStateA, epoch, Bits<T>::to(agg)));
    T excl = T(0);
    // Tile indices are below 2^24 (the launchers cap the grid), so 32-bit
    // signed arithmetic holds them and the walk past `first`.
    int32_t end = (int32_t)tile - 1;  // nearest predecessor not summed yet
    uint32_t spins = 0;
    while (true) {
        // K windows of 64 predecessors each, all loads in flight at once.
        uint64_t s[K], st[K];
#pragma unroll
        for (int k = 0; k < K; ++k) {
            const int32_t idx = end - lane - k * kWave;
            // Lanes past the segment start read an empty inclusive prefix; the
            // walk never sums them because `first` (always P) comes before them.
            s[k] = 0;
            st[k] = kStateP;
            if (idx >= (int32_t)first) {
                s[k] = status_load(status + idx);
                st[k] = status_state(s[k], epoch);
            }
        }
        bool done = false, retry = false;
#pragma unroll
        for (int k = 0; k < K; ++k) {
            if (done || retry) break;
            const uint64_t pmask = __ballot(st[k] == kStateP);
            const uint64_t xmask = __ballot(st[k] == kStateX);
            // lanes 0..p where p is the nearest predecessor with an inclusive prefix
            const uint64_t upto = pmask ? (((pmask & (~pmask + 1)) << 1) - 1) : ~0ull;
            if (xmask & upto) {  // a predecessor has not published: read again from here
                retry = true;
                break;
            }
            const T v = ((upto >> lane) & 1) ? Bits<T>::from((uint32_t)s[k]) : T(0);
            excl = excl + wave_sum(v);
            end -= kWave;
            done = pmask != 0;
        }
        if (done) break;
        if (retry) {
            if (++spins >= kSpinLimit) {
                if (lane == 0)
                    __hip_atomic_store(&h->error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                break;
            }
            __builtin_amdgcn_s_sleep(1);
        }
    }
    if (lane == 0) {
        adversarial_pause(tile ^ 0x5bd1e995u);
        status_store(status + tile, status_word(kStateP, epoch, Bits<T>::to(excl + agg)));
    }
    return excl;
}

// Called by one thread of every workgroup of a look-back launch after its
// last status access.  Only in the launch whose epoch is the last before the
// 30-bit status tag wraps does it do anything: the last workgroup to finish
// then zeroes every status word of the workspace, so that no word written
// 2^30 calls ago can ever be mistaken for a current one.
__device__ __forceinline__ void finish_epoch(WsHeader* h, uint32_t epoch, uint32_t nwg,
                                             uint64_t* status, int64_t status_words) {
    if ((epoch & kEpochMask) != kEpochMask) return;
    const uint32_t d = __hip_atomic_fetch_add(&h->done, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    if (d != nwg - 1) return;
    for (int64_t i = 0; i < status_words; ++i) status[i] = 0;
    __hip_atomic_store(&h->done, 0u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace ls
