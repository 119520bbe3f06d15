/*
 * libscan.h -- C ABI of libscan: device-wide prefix sums and scan-based
 * operators on one AMD MI355X (gfx950), hand-written HIP underneath.
 *
 * The operations follow "Parallel Scan on Ascend AI Accelerators"
 * (Wroblewski, Gottardo, Zouzias); each declaration names the passage that
 * defines what it computes.  How it is computed (single-pass decoupled
 * look-back over 64-lane wavefront tiles) is this library's own design.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Pointers named x, y, keys, mask, out, ... and every *_dev pointer are
 *    DEVICE pointers owned by the caller.  The library keeps no device memory
 *    of its own between calls and never allocates.
 *  - Arrays are dense and contiguous (row-major for rows x len matrices).
 *    Element alignment is enough; 16-byte aligned arrays take the vector path.
 *  - ws / ws_bytes: caller-owned device workspace of at least the size that
 *    libscan_workspace_bytes() reports for the op and sizes, 16-byte aligned.
 *    It must be zero-filled once before its first use (libscan_workspace_init
 *    does that; so does any zero fill) and afterwards be written only by
 *    libscan: every call leaves it ready for the next one, of any op, so it
 *    is never cleared again.  Calls that may run concurrently (on different
 *    streams) need distinct workspaces.
 *  - stream: a hipStream_t passed as void*; NULL is the null stream.  Calls
 *    only enqueue work: they return before the GPU finishes and never
 *    synchronise.  Counts and totals are written to device memory.
 *  - Integer sums wrap modulo 2^32 (two's complement).  Floating-point sums are
 *    accumulated in fp32 in an order that can vary from run to run.
 *  - Return value: LIBSCAN_OK, or a negative LIBSCAN_E* code for an argument
 *    or launch error; on error the outputs are unspecified.  Faults inside a
 *    kernel surface at the caller's next synchronisation, not here.
 *  - Argument checks (all before any HIP call): sizes must be >= 0; a NULL
 *    data pointer is accepted only when its size is 0; outputs may not
 *    partially overlap inputs (exact in-place is allowed where noted).
 */
#ifndef LIBSCAN_H
#define LIBSCAN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LIBSCAN_OK 0
#define LIBSCAN_EINVAL (-1)   /* invalid argument (size, NULL, overlap, alignment, parameter) */
#define LIBSCAN_ENOSPACE (-2) /* workspace smaller than libscan_workspace_bytes() */
#define LIBSCAN_EHIP (-3)     /* a HIP launch reported an error */
#define LIBSCAN_ERANGE (-4)   /* size beyond what the op supports */

/* Library version as MAJOR*10000 + MINOR*100 + PATCH. */
int libscan_version(void);

/* Static English text for a status code (never NULL). */
const char* libscan_status_string(int status);

/*
 * Zero-fill a workspace before its first use (enqueued on stream; a fill
 * kernel, not a memset, so it may be captured in a HIP graph).  ws must be
 * 16-byte aligned and ws_bytes a multiple of 8.
 */
int libscan_workspace_init(void* ws, size_t ws_bytes, void* stream);

/* Operation codes for libscan_workspace_bytes. */
#define LIBSCAN_OP_SCAN 1     /* every 1-D scan_* entry point (look-back) */
#define LIBSCAN_OP_SCAN_RSS 2 /* scan_inclusive_rss_* (reduce-then-scan) */

/*
 * Workspace size in bytes that op needs for n elements (rows/len/bits are
 * used by the row and sort ops and ignored otherwise).  Writes *bytes and
 * returns LIBSCAN_OK, or LIBSCAN_EINVAL for an unknown op / negative size /
 * NULL bytes, LIBSCAN_ERANGE if the sizes are beyond the op's limits.
 * Pure host function; needs no GPU.
 */
int libscan_workspace_bytes(int op, int64_t n, int64_t rows, int64_t len, int bits, size_t* bytes);

/* ------------------------------------------------------------------------
 * 1-D scans (Section 2: y_i = x_1 + ... + x_i; Appendix "Exclusive and
 * int8 scan": exclusive form y_0 = 0, y_i = x_1 + ... + x_{i-1}).
 * n >= 0 elements; at most 2^35 elements.  In-place (x == y) is allowed for
 * the same-type scans; any other overlap of x and y is LIBSCAN_EINVAL.
 * ------------------------------------------------------------------------ */
int scan_inclusive_i32(const int32_t* x, int32_t* y, int64_t n, void* ws, size_t ws_bytes,
                       void* stream);
int scan_exclusive_i32(const int32_t* x, int32_t* y, int64_t n, void* ws, size_t ws_bytes,
                       void* stream);
int scan_inclusive_f32(const float* x, float* y, int64_t n, void* ws, size_t ws_bytes,
                       void* stream);
int scan_exclusive_f32(const float* x, float* y, int64_t n, void* ws, size_t ws_bytes,
                       void* stream);

/* fp16 input (IEEE binary16 bit patterns), fp32 accumulation and output
 * (Section 3.1: the cube takes fp16 in and gives fp32 out; Section 6 scans
 * fp16).  x and y may not overlap. */
int scan_inclusive_f16f32(const uint16_t* x, float* y, int64_t n, void* ws, size_t ws_bytes,
                          void* stream);
int scan_exclusive_f16f32(const uint16_t* x, float* y, int64_t n, void* ws, size_t ws_bytes,
                          void* stream);

/* 8-bit input summed as unsigned byte values into int32 (Appendix
 * "Exclusive and int8 scan": int8 input, int32 accumulation; used on masks).
 * total_dev (nullable, device) receives the sum of all n bytes mod 2^32.
 * x and y may not overlap. */
int scan_exclusive_u8i32(const uint8_t* x, int32_t* y, int64_t n, int32_t* total_dev, void* ws,
                         size_t ws_bytes, void* stream);

/* Chunked scans (Section 6.1.1, "L2 cache splitting": consecutive chunks
 * scanned one after another, the last value of each carried into the next).
 * carry_in_dev (nullable, device, one element) is added in front of x, i.e.
 * y_i = carry + (x_1 + ... + x_i) for inclusive; total_out_dev (nullable,
 * device, one element) receives carry + (x_1 + ... + x_n), the carry for the
 * next chunk.  carry_in_dev and total_out_dev may be the same pointer. */
int scan_inclusive_i32_carry(const int32_t* x, int32_t* y, int64_t n, const int32_t* carry_in_dev,
                             int32_t* total_out_dev, void* ws, size_t ws_bytes, void* stream);
int scan_exclusive_i32_carry(const int32_t* x, int32_t* y, int64_t n, const int32_t* carry_in_dev,
                             int32_t* total_out_dev, void* ws, size_t ws_bytes, void* stream);
int scan_inclusive_f32_carry(const float* x, float* y, int64_t n, const float* carry_in_dev,
                             float* total_out_dev, void* ws, size_t ws_bytes, void* stream);
int scan_exclusive_f32_carry(const float* x, float* y, int64_t n, const float* carry_in_dev,
                             float* total_out_dev, void* ws, size_t ws_bytes, void* stream);

/* Reduce-then-scan check variant (Section 2.1, the Reduce-Scan-Scan strategy;
 * the two phases of Algorithm 3, MCScan): per-tile reductions, one scan of
 * the tile sums, then every tile rescanned with its carry.  Reads x twice.
 * Same result definition and arguments as scan_inclusive_i32 / _f32
 * (workspace: LIBSCAN_OP_SCAN_RSS). */
int scan_inclusive_rss_i32(const int32_t* x, int32_t* y, int64_t n, void* ws, size_t ws_bytes,
                           void* stream);
int scan_inclusive_rss_f32(const float* x, float* y, int64_t n, void* ws, size_t ws_bytes,
                           void* stream);

#ifdef __cplusplus
}
#endif

#endif /* LIBSCAN_H */
