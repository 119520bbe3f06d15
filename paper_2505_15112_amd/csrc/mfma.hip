// mfma.hip -- the tile-local scan on the matrix cores (Section 4.1, ScanU),
// for fp16 input with fp32 accumulation and output.
//
// ScanU views a tile of s*s elements as a row-major s x s matrix A and takes
// the row scans with one matrix product, A * U_s (U_s upper triangular,
// ones on and above the diagonal: (A U_s)[i][j] = A[i][0] + ... + A[i][j]);
// the vector unit then adds to every row the sum of the rows before it and
// the carry of the tiles before.  Here s = 32: a 1024-element block is one
// v_mfma_f32_32x32x16_f16 pair (k = 0..15 and 16..31), products are exact
// (x * 1 or x * 0) and the sums are fp32.  The row totals (column 31 of the
// product) are scanned across the wave by DPP, and the blocks, waves and
// tiles are chained exactly as in the wavefront scan (running sum over the
// wave's blocks, wave totals through LDS, decoupled look-back).
//
// Operand layouts of the 32x32x16 fp16 MFMA (lane l, 64 lanes): A gives lane
// l the 8 elements A[l % 32][8 (l / 32) + t]; B gives it B[8 (l / 32) + t]
// [l % 32]; the 16 accumulators of lane l hold D[8 (r / 4) + 4 (l / 32) +
// r % 4][l % 32], r = 0..15.
//
// Measured against the wavefront tiles of the same size (rocprofv3 kernel
// trace, MI355X): 332 against 350 us at n = 2^28, 30.2 against 31.7 us at
// 2^24 from cold caches, so inclusive fp16 scans use it by default.  The
// scan is bound by HBM either way; this kernel loads 16 bytes per lane per
// matrix operand where the wavefront tile loads 8, and its accumulators leave
// as 4-byte stores of one matrix column each.  Whole 32768-element tiles run
// here; a ragged tail (fewer than 32768 elements) is scanned by the
// wavefront kernel with this launch's total as its carry.  A tile holding an
// infinity or a NaN is scanned on the vector units (IEEE propagation: the
// matrix product would multiply it by the zeros of U_s).
#include "launch.hpp"
#include "tile.hpp"

namespace ls {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kS = 32;                 // matrix side
constexpr int kBlock = kS * kS;        // elements per matrix block
constexpr int kMfmaBlocks = 4;         // blocks per wave
constexpr int kMfmaWaves = 8;          // waves per workgroup
constexpr int64_t kMfmaTile = (int64_t)kMfmaWaves * kMfmaBlocks * kBlock;  // 32768 elements
static_assert(kMfmaTile == kMfmaTileElems, "tile size seen by the dispatcher");

// Half h of U_s as the B operand: rows k = 16h + 8 (l / 32) + t, column l % 32.
__device__ __forceinline__ h8 upper_ones(int h) {
    const int lane = lane_id();
    const int j = lane & (kS - 1), k0 = 16 * h + 8 * (lane >> 5);
    h8 u;
#pragma unroll
    for (int t = 0; t < 8; ++t) u[t] = (k0 + t <= j) ? (_Float16)1.0f : (_Float16)0.0f;
    return u;
}

// Half h of the (complete, 16-byte aligned) block at xb as the A operand.
__device__ __forceinline__ h8 load_half(const uint16_t* xb, int h) {
    const int lane = lane_id();
    const int off = (lane & (kS - 1)) * kS + 16 * h + 8 * (lane >> 5);
    return __builtin_bit_cast(h8, *reinterpret_cast<const u32x4*>(xb + off));
}

// True if any of the 8 fp16 values is an infinity or a NaN (exponent bits
// all ones).
__device__ __forceinline__ bool has_special(h8 v) {
    const u32x4 r = __builtin_bit_cast(u32x4, v);
    bool s = false;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const uint32_t e = r[q] & 0x7C007C00u;
        s |= (e & 0xFFFFu) == 0x7C00u || (e >> 16) == 0x7C00u;
    }
    return s;
}

// A whole tile on the vector units: eight passes of 4096 elements (the
// wavefront tile scan), swept twice -- the tile's sum for the look-back,
// then the outputs with the carry -- with the pass sums taken the same way
// both times.  Used for tiles holding an infinity or a NaN.
__device__ __forceinline__ void mfma_tile_on_vector_units(
    const uint16_t* x, float* y, int64_t tbase, uint32_t tile32, uint32_t epoch, WsHeader* hdr,
    uint64_t* status, int64_t status_words, uint32_t ntiles, float* total_out, float* s_wtot,
    float* s_carry) {
    using P = Tile<uint16_t, float, 4, 2, kMfmaWaves>;
    constexpr int kPasses = (int)(kMfmaTile / P::kElems);
    const int64_t tend = tbase + kMfmaTile;
    float agg = 0.f;
    for (int q = 0; q < kPasses; ++q) {
        float v[P::J][P::V];
        P::template load<true>(x, tend, tbase + q * P::kElems, v);
        float wofs;
        agg = agg + P::combine_waves(P::template wave_scan<false>(v), s_wtot, &wofs);
        __syncthreads();  // s_wtot is rewritten by the next pass
    }
    if (threadIdx.x < kWave) {
        const float excl = lookback<float>(status, tile32, 0u, agg, 0.f, epoch, hdr);
        if (threadIdx.x == 0) {
            *s_carry = excl;
            if (total_out && tile32 == ntiles - 1) *total_out = excl + agg;
            finish_epoch(hdr, epoch, ntiles, status, status_words);
        }
    }
    __syncthreads();
    float carry = *s_carry;
    for (int q = 0; q < kPasses; ++q) {
        float v[P::J][P::V];
        const int64_t base = tbase + q * P::kElems;
        P::template load<true>(x, tend, base, v);
        float wofs;
        const float pagg = P::combine_waves(P::template wave_scan<false>(v), s_wtot, &wofs);
        P::template store<true>(y, tend, base, v, carry + wofs);
        carry = carry + pagg;
        __syncthreads();
    }
}

// Full tiles only (the launcher scans a ragged tail with the wavefront
// kernel, carrying this launch's total); x 16-byte aligned.  The last tile
// writes the total to *total_out when total_out is not null.
__global__ __launch_bounds__(kMfmaWaves * kWave) LS_OCCUPANCY4 void k_scan_mfma_f16(
    const uint16_t* x, float* y, WsHeader* hdr, uint64_t* status, int64_t status_words,
    uint32_t ntiles, float* total_out) {
    __shared__ Ticket s_ticket;
    __shared__ float s_wtot[kMfmaWaves];
    __shared__ float s_carry;
    __shared__ __attribute__((aligned(16))) float s_row[kMfmaWaves][kS];  // per wave: row totals, then row prefixes

    if (threadIdx.x == 0) s_ticket = take_ticket(hdr, ntiles);
    __syncthreads();
    const uint32_t tile32 = (uint32_t)__builtin_amdgcn_readfirstlane(s_ticket.tile);
    const uint32_t epoch = (uint32_t)__builtin_amdgcn_readfirstlane(s_ticket.epoch);
    if (tile32 >= ntiles) {  // only with a workspace that was never zero-filled
        if (threadIdx.x == 0)
            __hip_atomic_store(&hdr->error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return;
    }
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int lane = lane_id();
    const int64_t wbase = (int64_t)tile32 * kMfmaTile + (int64_t)w * kMfmaBlocks * kBlock;

    h8 a[kMfmaBlocks][2];
#pragma unroll
    for (int b = 0; b < kMfmaBlocks; ++b)
#pragma unroll
        for (int h = 0; h < 2; ++h) a[b][h] = load_half(x + wbase + b * kBlock, h);

    // An infinity or a NaN would meet the zeros of U_32 (inf * 0 is NaN) and
    // spoil the sums of the elements before it: such a tile (uniform: one
    // vote per workgroup) is scanned on the vector units instead.
    bool special = false;
#pragma unroll
    for (int b = 0; b < kMfmaBlocks; ++b)
#pragma unroll
        for (int h = 0; h < 2; ++h) special |= has_special(a[b][h]);
    if (__syncthreads_or(special)) {
        mfma_tile_on_vector_units(x, y, (int64_t)tile32 * kMfmaTile, tile32, epoch, hdr, status,
                                  status_words, ntiles, total_out, s_wtot, &s_carry);
        return;
    }

    // Block by block: the row scans on the matrix cores (acc[b] = A_b * U_32),
    // then every row gets the rows before it and the wave's earlier blocks.
    const h8 u0 = upper_ones(0), u1 = upper_ones(1);
    f32x16 acc[kMfmaBlocks];
    float* rowt = s_row[w];
    const int half = lane >> 5;  // which 4 of every 8 rows this lane's accumulators hold
    float run = 0.f;
#pragma unroll
    for (int b = 0; b < kMfmaBlocks; ++b) {
        const f32x16 zero = {};
        acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a[b][0], u0, zero, 0, 0, 0);
        acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a[b][1], u1, acc[b], 0, 0, 0);
        if ((lane & (kS - 1)) == kS - 1) {  // column 31 holds the row totals
#pragma unroll
            for (int r = 0; r < 16; ++r) rowt[8 * (r >> 2) + 4 * half + (r & 3)] = acc[b][r];
        }
        wave_lds_sync();
        const float t = lane < kS ? rowt[lane] : 0.f;
        const float inc = wave_incl_scan(t);
        const float before = wave_shr1(inc);  // lane i < 32: rows 0..i-1 of the block
        const float btot = lane_read(inc, kS - 1);
        wave_lds_sync();
        if (lane < kS) rowt[lane] = run + before;
        wave_lds_sync();
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const f32x4 pr = *reinterpret_cast<const f32x4*>(rowt + 8 * q + 4 * half);
#pragma unroll
            for (int e = 0; e < 4; ++e) acc[b][4 * q + e] = pr[e] + acc[b][4 * q + e];
        }
        // Make the sums here: left to itself the compiler defers them to the
        // stores and keeps the row prefixes live (in scratch) meanwhile.
        asm volatile("" : "+v"(acc[b]));
        run = run + btot;
        wave_lds_sync();  // rowt is rewritten by the next block
    }

    float wofs;
    const float agg = Tile<float, float, 4, 1, kMfmaWaves>::combine_waves(run, s_wtot, &wofs);
    if (threadIdx.x < kWave) {
        const float excl = lookback<float>(status, tile32, 0u, agg, 0.f, epoch, hdr);
        if (threadIdx.x == 0) {
            s_carry = excl;
            if (total_out && tile32 == ntiles - 1) *total_out = excl + agg;
            finish_epoch(hdr, epoch, ntiles, status, status_words);
        }
    }
    __syncthreads();
    const float carry = s_carry + wofs;
    const int j = lane & (kS - 1);
#pragma unroll
    for (int b = 0; b < kMfmaBlocks; ++b) {
        float* yb = y + wbase + b * kBlock;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int i = 8 * (r >> 2) + 4 * half + (r & 3);
            __builtin_nontemporal_store(carry + acc[b][r], yb + i * kS + j);
        }
    }
}

// ---------------------------------------------------------------- bytes
//
// The exclusive byte scan (appendix "Exclusive and int8 scan": int8 in,
// int32 sums) the same way, on v_mfma_i32_32x32x32_i8: a 1024-byte block
// is one product with the strictly upper triangular U' (U'[k][j] = 1 for
// k < j), whose entry (i, j) is the sum of row i before column j.  The MFMA
// multiplies signed bytes, so it is fed x - 128 (the byte with its top bit
// flipped) and 128 j is added back to column j: exact in 32-bit integers.
// The row totals need no product: each lane sums its 16 bytes with
// v_dot4_u32_u8 and adds the lane holding the other half of the row.
// Measured against the wavefront byte tiles: 251 against 251 us at
// n = 2^28 -- a tie, so the default byte scan stays on the wavefront tiles
// and this kernel is reached through scan_exclusive_u8i32_mfma only.
// Operand layout: A gives lane l the 16 bytes A[l % 32][16 (l / 32) + t],
// B gives it B[16 (l / 32) + t][l % 32]; the accumulators are laid out as
// for the fp16 product.
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ i32x4 strict_upper_ones_i8() {
    const int lane = lane_id();
    const int j = lane & (kS - 1), k0 = 16 * (lane >> 5);
    uint32_t w[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        w[q] = 0;
#pragma unroll
        for (int t = 0; t < 4; ++t) w[q] |= (uint32_t)(k0 + 4 * q + t < j) << (8 * t);
    }
    return i32x4{(int)w[0], (int)w[1], (int)w[2], (int)w[3]};
}

__global__ __launch_bounds__(kMfmaWaves * kWave) LS_OCCUPANCY4 void k_scan_mfma_u8(
    const uint8_t* x, uint32_t* y, WsHeader* hdr, uint64_t* status, int64_t status_words,
    uint32_t ntiles, uint32_t* total_out) {
    __shared__ Ticket s_ticket;
    __shared__ uint32_t s_wtot[kMfmaWaves];
    __shared__ uint32_t s_carry;
    __shared__ __attribute__((aligned(16))) uint32_t s_row[kMfmaWaves][kS];  // per wave: row prefixes

    if (threadIdx.x == 0) s_ticket = take_ticket(hdr, ntiles);
    __syncthreads();
    const uint32_t tile32 = (uint32_t)__builtin_amdgcn_readfirstlane(s_ticket.tile);
    const uint32_t epoch = (uint32_t)__builtin_amdgcn_readfirstlane(s_ticket.epoch);
    if (tile32 >= ntiles) {  // only with a workspace that was never zero-filled
        if (threadIdx.x == 0)
            __hip_atomic_store(&hdr->error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return;
    }
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int lane = lane_id();
    const int64_t wbase = (int64_t)tile32 * kMfmaTile + (int64_t)w * kMfmaBlocks * kBlock;
    const int aoff = (lane & (kS - 1)) * kS + 16 * (lane >> 5);

    u32x4 a[kMfmaBlocks];
#pragma unroll
    for (int b = 0; b < kMfmaBlocks; ++b)
        a[b] = *reinterpret_cast<const u32x4*>(x + wbase + b * kBlock + aoff);

    const i32x4 us = strict_upper_ones_i8();
    const uint32_t colfix = 128u * (uint32_t)(lane & (kS - 1));  // 128 j
    i32x16 acc[kMfmaBlocks];
    uint32_t* rowt = s_row[w];
    const int half = lane >> 5;
    uint32_t run = 0;
#pragma unroll
    for (int b = 0; b < kMfmaBlocks; ++b) {
        const u32x4 sgn = a[b] ^ 0x80808080u;  // x - 128 as signed bytes
        const i32x16 zero = {};
        acc[b] = __builtin_amdgcn_mfma_i32_32x32x32_i8(__builtin_bit_cast(i32x4, sgn), us, zero,
                                                       0, 0, 0);
        // row totals: this lane's 16 bytes, plus the other half of the row
        uint32_t sum = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) sum = __builtin_amdgcn_udot4(a[b][q], 0x01010101u, sum, false);
        const uint32_t t = sum + (uint32_t)__shfl_xor((int)sum, 32);
        const uint32_t inc = wave_incl_scan(lane < kS ? t : 0u);
        const uint32_t before = wave_shr1(inc);  // lane i < 32: rows 0..i-1 of the block
        const uint32_t btot = lane_read(inc, kS - 1);
        if (lane < kS) rowt[lane] = run + before;
        wave_lds_sync();
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const u32x4 pr = *reinterpret_cast<const u32x4*>(rowt + 8 * q + 4 * half);
#pragma unroll
            for (int e = 0; e < 4; ++e)
                acc[b][4 * q + e] = (int)((uint32_t)acc[b][4 * q + e] + colfix + pr[e]);
        }
        asm volatile("" : "+v"(acc[b]));
        run = run + btot;
        wave_lds_sync();  // rowt is rewritten by the next block
    }

    uint32_t wofs;
    const uint32_t agg =
        Tile<uint32_t, uint32_t, 4, 1, kMfmaWaves>::combine_waves(run, s_wtot, &wofs);
    if (threadIdx.x < kWave) {
        const uint32_t excl = lookback<uint32_t>(status, tile32, 0u, agg, 0u, epoch, hdr);
        if (threadIdx.x == 0) {
            s_carry = excl;
            if (total_out && tile32 == ntiles - 1) *total_out = excl + agg;
            finish_epoch(hdr, epoch, ntiles, status, status_words);
        }
    }
    __syncthreads();
    const uint32_t carry = s_carry + wofs;
    const int j = lane & (kS - 1);
#pragma unroll
    for (int b = 0; b < kMfmaBlocks; ++b) {
        uint32_t* yb = y + wbase + b * kBlock;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int i = 8 * (r >> 2) + 4 * half + (r & 3);
            __builtin_nontemporal_store(carry + (uint32_t)acc[b][r], yb + i * kS + j);
        }
    }
}

hipError_t launch_scan1d_mfma_u8(const uint8_t* x, uint32_t* y, int64_t n, uint32_t* total_out,
                                 void* ws, size_t ws_bytes, hipStream_t stream) {
    WsHeader* hdr = reinterpret_cast<WsHeader*>(ws);
    uint64_t* status = reinterpret_cast<uint64_t*>(reinterpret_cast<char*>(ws) + kWsHeader);
    const int64_t status_words = (int64_t)((ws_bytes - kWsHeader) / sizeof(uint64_t));
    const int64_t full = n / kMfmaTile, done = full * kMfmaTile;
    uint32_t* carry = reinterpret_cast<uint32_t*>(&hdr->reserved[0]);
    if (full > 0)
        hipLaunchKernelGGL(k_scan_mfma_u8, dim3((unsigned)full), dim3(kMfmaWaves * kWave), 0,
                           stream, x, y, hdr, status, status_words, (uint32_t)full,
                           done < n ? carry : total_out);
    if (done < n)
        return launch_scan1d_tiles(Kind::U8I32, true, x + done, y + done, n - done,
                                   full > 0 ? carry : nullptr, total_out, ws, ws_bytes, stream);
    return hipGetLastError();
}

hipError_t launch_scan1d_mfma_f16(const uint16_t* x, float* y, int64_t n, void* ws,
                                  size_t ws_bytes, hipStream_t stream) {
    WsHeader* hdr = reinterpret_cast<WsHeader*>(ws);
    uint64_t* status = reinterpret_cast<uint64_t*>(reinterpret_cast<char*>(ws) + kWsHeader);
    const int64_t status_words = (int64_t)((ws_bytes - kWsHeader) / sizeof(uint64_t));
    const int64_t full = n / kMfmaTile, done = full * kMfmaTile;
    // the first launch's total, read by the tail's launch (a header word no
    // kernel else uses; the two launches are ordered on the stream)
    float* carry = reinterpret_cast<float*>(&hdr->reserved[0]);
    if (full > 0)
        hipLaunchKernelGGL(k_scan_mfma_f16, dim3((unsigned)full), dim3(kMfmaWaves * kWave), 0,
                           stream, x, y, hdr, status, status_words, (uint32_t)full,
                           done < n ? carry : nullptr);
    if (done < n)
        return launch_scan1d_tiles(Kind::F16F32, false, x + done, y + done, n - done,
                                   full > 0 ? carry : nullptr, nullptr, ws, ws_bytes, stream);
    return hipGetLastError();
}

}  // namespace ls
