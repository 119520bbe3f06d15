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
 *    DEVICE pointers owned by the caller.  The library never allocates;
 *    its only device memory is the static workspace of
 *    scan_inclusive_i32_noalloc.
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
 *    accumulated in fp32 in an order that can vary from run to run;
 *    infinities and NaNs propagate as in IEEE arithmetic (a running sum is
 *    NaN once a NaN or both infinities precede it), whatever the order.
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

/*
 * The workspace's error word (Section 2.1's decoupled look-back waits on
 * other workgroups; here every such wait is bounded).  Kernels set it to 1,
 * and carry on with unspecified outputs instead of hanging, when a bounded
 * wait for another workgroup gives up or a tile ticket lies outside the
 * launch: what a workspace that was not zero-filled before its first use,
 * was written by something other than libscan, or was shared by calls that
 * ran concurrently leads to.  It stays set until reset.  This enqueues on
 * stream a copy of the word into error_dev (device, one int32: 0 = every call
 * since the last reset ran its protocol to the end) and, when reset != 0,
 * clears it; it allocates nothing and does not synchronise (read error_dev
 * after the stream has reached it).  ws 16-byte aligned and at least 256
 * bytes (LIBSCAN_ENOSPACE otherwise), error_dev 4-byte aligned and outside
 * the workspace header, else LIBSCAN_EINVAL.
 */
int libscan_workspace_error(void* ws, size_t ws_bytes, int32_t* error_dev, int reset,
                            void* stream);

/* Operation codes for libscan_workspace_bytes. */
#define LIBSCAN_OP_SCAN 1     /* every 1-D scan_* entry point (look-back) */
#define LIBSCAN_OP_SCAN_RSS 2 /* scan_inclusive_rss_* (reduce-then-scan) */
#define LIBSCAN_OP_SCAN_ROWS 3 /* scan_rows_* and topp_cutoff_f32 (rows, len) */
#define LIBSCAN_OP_COMPACT 4   /* compact_by_mask_f32 and split_by_flags_u32 (n) */
#define LIBSCAN_OP_RADIX_SORT 5 /* radix_sort_u32 (n, bits = bits_per_pass); typed sorts (bits = 8) */
#define LIBSCAN_OP_SORT_ROWS 6  /* radix_sort_rows_f32 (rows, len) */
#define LIBSCAN_OP_WEIGHTED_SAMPLE 7 /* weighted_sample_f32 (rows, len) */
#define LIBSCAN_OP_TOPP_SAMPLE 8 /* topp_sample_f32 (rows, len) */
#define LIBSCAN_OP_TOPK 9       /* topk_rows_f32 (rows, len, n = k) */

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
 * fp16).  x and y may not overlap.  The inclusive scan of a 16-byte aligned
 * x with n >= 2^27 takes its tile-local scans on the matrix cores (see
 * scan_inclusive_f16f32_mfma), otherwise the wavefront tiles. */
int scan_inclusive_f16f32(const uint16_t* x, float* y, int64_t n, void* ws, size_t ws_bytes,
                          void* stream);
int scan_exclusive_f16f32(const uint16_t* x, float* y, int64_t n, void* ws, size_t ws_bytes,
                          void* stream);

/* The same inclusive fp16 -> fp32 scan with the tile-local scan on the
 * matrix cores, as ScanU does it (Section 4.1, Algorithm 1): every block of
 * 32 x 32 elements, viewed as a row-major matrix A, gives its row scans as
 * A * U_32 (U_32 upper triangular ones) on v_mfma_f32_32x32x16_f16; rows,
 * blocks and tiles are then chained as in scan_inclusive_f16f32.  Same
 * arguments, workspace (LIBSCAN_OP_SCAN) and error behaviour, except that x
 * must be 16-byte aligned (one matrix operand is one 16-byte load per lane)
 * and y 4-byte aligned, else LIBSCAN_EINVAL; x and y may not overlap.  Whole
 * 32768-element tiles take the matrix-core kernel, a shorter tail the
 * wavefront one.  Results agree with the wavefront scan within the float
 * tolerance (exactly on {-1, 0, 1} inputs); measured faster than it from
 * n = 2^27 on (slower below), which is why scan_inclusive_f16f32 uses this
 * path for such arrays.  A tile holding
 * an infinity or a NaN is scanned on the vector units instead (in the
 * product it would meet the zeros of U_32, and inf * 0 is NaN). */
int scan_inclusive_f16f32_mfma(const uint16_t* x, float* y, int64_t n, void* ws,
                               size_t ws_bytes, void* stream);

/* The inclusive fp16 -> fp32 scan on the wavefront tiles only (lane-serial,
 * DPP and LDS tile scan), whatever n and the alignment: the baseline the
 * matrix-core path is measured against.  Arguments and errors as
 * scan_inclusive_f16f32. */
int scan_inclusive_f16f32_wave(const uint16_t* x, float* y, int64_t n, void* ws,
                               size_t ws_bytes, void* stream);

/* 8-bit input summed as unsigned byte values into int32 (Appendix
 * "Exclusive and int8 scan": int8 input, int32 accumulation; used on masks).
 * total_dev (nullable, device) receives the sum of all n bytes mod 2^32.
 * x and y may not overlap. */
int scan_exclusive_u8i32(const uint8_t* x, int32_t* y, int64_t n, int32_t* total_dev, void* ws,
                         size_t ws_bytes, void* stream);

/* The same exclusive byte scan with the tile-local scans on the matrix cores
 * (Section 4.1's ScanU with the strictly upper triangular ones matrix, which
 * gives exclusive row scans directly): each block of 32 x 32 bytes is one
 * v_mfma_i32_32x32x32_i8 product on x - 128 (the signed form of the byte),
 * corrected by 128 j per column j, exact in int32.  x must be 16-byte aligned
 * and y 4-byte aligned (else LIBSCAN_EINVAL); otherwise as
 * scan_exclusive_u8i32.  Whole 32768-byte tiles run on the matrix cores, a
 * shorter tail on the wavefront tiles.  Measured no faster than the
 * wavefront tiles, so scan_exclusive_u8i32 does not use it; kept as the
 * measured alternative. */
int scan_exclusive_u8i32_mfma(const uint8_t* x, int32_t* y, int64_t n, int32_t* total_dev,
                              void* ws, size_t ws_bytes, void* stream);

/* The exclusive byte scan on the wavefront tiles only (any n, any
 * alignment), which is what scan_exclusive_u8i32 runs: the baseline the
 * matrix-core path is measured against. */
int scan_exclusive_u8i32_wave(const uint8_t* x, int32_t* y, int64_t n, int32_t* total_dev,
                              void* ws, size_t ws_bytes, void* stream);

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

/* ------------------------------------------------------------------------
 * Batched scans (appendix "Multiple (Batched) Scans"): every row of the
 * row-major rows x len matrix x is scanned on its own (inclusive, or
 * exclusive when `exclusive` != 0) into y of the same layout.  In-place
 * (x == y) is allowed.  rows * len <= 2^35 and rows * ceil(len / 4096) <=
 * 2^24.  Workspace: LIBSCAN_OP_SCAN_ROWS with (rows, len).
 * ------------------------------------------------------------------------ */
int scan_rows_i32(const int32_t* x, int32_t* y, int64_t rows, int64_t len, int exclusive, void* ws,
                  size_t ws_bytes, void* stream);
int scan_rows_f32(const float* x, float* y, int64_t rows, int64_t len, int exclusive, void* ws,
                  size_t ws_bytes, void* stream);

/* Top-p (nucleus) cutoff (Section 5 "Top-p or Nucleus Sampling": sort, then
 * cumulative sum, then cut at p).  probs: rows x len, every row already sorted
 * in descending order.  cutoff (device, rows int32) receives, per row, the
 * smallest 0-based index i with probs[r][0] + ... + probs[r][i] >= p, the
 * running sum taken in fp32; len - 1 if no prefix reaches p (so p <= 0 gives
 * 0 for non-negative rows); -1 for len == 0.  Tokens 0..cutoff[r] are kept.
 * p must not be NaN; len <= INT32_MAX.  Workspace: LIBSCAN_OP_SCAN_ROWS. */
int topp_cutoff_f32(const float* probs, int32_t* cutoff, int64_t rows, int64_t len, float p,
                    void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Scan-based data movement (Section 5).  n <= INT32_MAX (positions, counts
 * and indices are int32).  No output may overlap any input or another
 * output.  Workspace: LIBSCAN_OP_COMPACT with n.
 * ------------------------------------------------------------------------ */

/* Compress (Section 5 "Compress", i.e. torch.masked_select): out receives the
 * x_i whose mask byte is non-zero, in index order, as bit copies; idx_out
 * (nullable) their source indices; count_dev (device, one int32, required)
 * their number.  out and idx_out need room for n elements (only the first
 * count are written).  Single pass: mask and x read once. */
int compact_by_mask_f32(const float* x, const uint8_t* mask, float* out, int32_t* idx_out,
                        int32_t* count_dev, int64_t n, void* ws, size_t ws_bytes, void* stream);

/* Split (Section 5 "Split", the SplitInd operator): a stable partition of keys
 * -- every key whose flag byte is non-zero first, then all the others, each
 * group in index order.  idx_out (nullable) receives idx_in[i] of every moved
 * key, or i when idx_in is NULL; n_true_dev (nullable, device, one int32) the
 * number of flagged keys. */
int split_by_flags_u32(const uint32_t* keys, const int32_t* idx_in, const uint8_t* flags,
                       uint32_t* keys_out, int32_t* idx_out, int32_t* n_true_dev, int64_t n,
                       void* ws, size_t ws_bytes, void* stream);

/* LSD radix sort (Section 5 "Radix Sort": a loop over the key bits from the
 * least significant one, each step a stable split; Section 6 returns source
 * indices like PyTorch's sort()).  keys_out receives the n keys in ascending
 * order, stably; perm_out (nullable) the source index of each, so that
 * keys_out[i] == keys[perm_out[i]].  bits_per_pass: 1 (32 split passes), 4
 * (8 passes of 16-way stable splits) or 8 (4 passes of 256-way stable
 * splits); all give the same output.  keys_tmp
 * (and perm_tmp when perm_out is given) are caller-provided n-element
 * ping-pong buffers whose contents are clobbered.  No two of keys, keys_out,
 * perm_out, keys_tmp, perm_tmp may overlap.  n <= INT32_MAX.  Workspace:
 * LIBSCAN_OP_RADIX_SORT with n and bits = bits_per_pass. */
int radix_sort_u32(const uint32_t* keys, uint32_t* keys_out, int32_t* perm_out, uint32_t* keys_tmp,
                   int32_t* perm_tmp, int64_t n, int bits_per_pass, void* ws, size_t ws_bytes,
                   void* stream);

/* LSD radix sort of signed and floating-point keys (Section 5 "Radix Sort":
 * the keys are encoded so that an unsigned sort orders them -- the most
 * significant bit of non-negative numbers and every bit of negative ones
 * inverted; for two's-complement integers only the sign bit -- and decoded
 * afterwards; the paper sorts fp16 this way).  Here the encoding is applied
 * by the first pass's loads and undone by the last pass's stores, with 8-bit
 * digits: 4 passes for 32-bit keys, 2 for fp16.  descending != 0 sorts in
 * descending order (the code inverted).  Stable either way: ties keep index
 * order.  Floats follow IEEE 754 totalOrder, the order the encoding gives
 * every bit pattern: -NaN < -Inf < ... < -0 < +0 < ... < +Inf < +NaN.
 * keys_out, perm_out (nullable: keys only), keys_tmp and perm_tmp as in
 * radix_sort_u32 (elements of the key type; no two may overlap).
 * n <= INT32_MAX.  Workspace: LIBSCAN_OP_RADIX_SORT with n and bits = 8. */
int radix_sort_i32(const int32_t* keys, int32_t* keys_out, int32_t* perm_out, int32_t* keys_tmp,
                   int32_t* perm_tmp, int64_t n, int descending, void* ws, size_t ws_bytes,
                   void* stream);
int radix_sort_f32(const float* keys, float* keys_out, int32_t* perm_out, float* keys_tmp,
                   int32_t* perm_tmp, int64_t n, int descending, void* ws, size_t ws_bytes,
                   void* stream);
int radix_sort_f16(const uint16_t* keys, uint16_t* keys_out, int32_t* perm_out, uint16_t* keys_tmp,
                   int32_t* perm_tmp, int64_t n, int descending, void* ws, size_t ws_bytes,
                   void* stream);

/* Batched sort (Section 5 "Radix Sort" applied to each row, as the top-p
 * sampler needs it): each of the rows x len rows of fp32 keys sorted on its
 * own, stably, ascending or (descending != 0) descending, in IEEE 754
 * totalOrder as radix_sort_f32.  perm_out (nullable) receives each key's index
 * within its row (0..len-1).  keys_tmp / perm_tmp are rows x len ping-pong
 * buffers.  No two of keys, keys_out, perm_out, keys_tmp, perm_tmp may
 * overlap.  rows * len <= INT32_MAX and rows * ceil(len / 8192) <= 2^24.
 * Workspace: LIBSCAN_OP_SORT_ROWS with (rows, len). */
int radix_sort_rows_f32(const float* keys, float* keys_out, int32_t* perm_out, float* keys_tmp,
                        int32_t* perm_tmp, int64_t rows, int64_t len, int descending, void* ws,
                        size_t ws_bytes, void* stream);

/* Weighted sampling by inverse transform (Appendix "Weighted Sampling": a scan
 * of the weights, then the first index whose running sum exceeds theta times
 * the total).  w: rows x len non-negative fp32 weights; theta_dev (device,
 * rows floats, each in [0, 1)) the uniform draws; out (device, rows int32)
 * receives per row the smallest 0-based i with w[r][0] + ... + w[r][i] >
 * theta[r] * (w[r][0] + ... + w[r][len-1]), the sums taken in fp32; len - 1
 * when rounding leaves no such i; -1 for len == 0.  Index i is drawn with
 * probability w[r][i] / total when theta is uniform.  Any row length
 * (len <= INT32_MAX, limits as scan_rows).  No output may overlap an input.
 * Workspace: LIBSCAN_OP_WEIGHTED_SAMPLE with (rows, len). */
int weighted_sample_f32(const float* w, const float* theta_dev, int32_t* out, int64_t rows,
                        int64_t len, void* ws, size_t ws_bytes, void* stream);

/* Top-p (nucleus) sampling on unsorted rows (Section 5 "Top-p or Nucleus
 * Sampling": sort each row in descending order keeping the token indices,
 * take the running sum, cut at p, draw from what is kept).  probs: rows x len
 * non-negative fp32 probabilities (any order; they need not sum to 1).  Per
 * row: the stable descending sort S (ties keep index order), the cutoff k as
 * topp_cutoff_f32 computes it on S, then the draw by inverse transform over
 * S[0..k]: the smallest j <= k with S[0] + ... + S[j] > theta[r] * C, where C
 * is the running sum at k (fp32; j = k when rounding leaves none).
 * token_out (device, rows int32) receives the token index of S[j] in the
 * original row; cutoff_out (nullable, device, rows int32) receives k.  Both
 * are -1 for len == 0.  theta_dev as in weighted_sample_f32; p must not be
 * NaN.  rows * len <= INT32_MAX, rows * ceil(len / 8192) <= 2^24.
 * scratch: caller device memory, 16-byte aligned, of at least
 * libscan_scratch_bytes(LIBSCAN_OP_TOPP_SAMPLE, rows, len, 0) bytes (16 per
 * element: the sorted copies and the sort's ping-pong buffers).  Unlike the
 * workspace it needs no initialisation and carries nothing between calls; it
 * is clobbered and may not overlap any input, output or the workspace.
 * Workspace: LIBSCAN_OP_TOPP_SAMPLE with (rows, len). */
int topp_sample_f32(const float* probs, const float* theta_dev, float p, int32_t* token_out,
                    int32_t* cutoff_out, int64_t rows, int64_t len, void* scratch,
                    size_t scratch_bytes, void* ws, size_t ws_bytes, void* stream);

/* Top-k of every row (Section 5 "Top-k": selection, a partial quicksort, on
 * stable splits).  x: rows x len fp32.  Per row, values_out receives the k
 * largest values (largest != 0) or the k smallest, in IEEE 754 totalOrder
 * (as radix_sort_f32: +NaN is the largest value, -NaN the smallest), listed
 * in descending (ascending) order, equal values by increasing index: the
 * first k entries of the row's stable sort in that direction, as bit
 * copies; idx_out receives their indices within the row.  values_out and
 * idx_out are rows x k.  0 <= k <= len (EINVAL otherwise); len <= INT32_MAX,
 * rows * ceil(len / 4096) <= 2^24, rows * k <= INT32_MAX.  Rows of at most
 * 2^17 elements with k <= 256: each tile of the row (8192 elements, 4096
 * for rows of at most 16384) keeps its keys whose top 16 bits are at least
 * those of its own k-th largest, and one workgroup per row selects the k
 * largest of those and places them by rank (one read of the row; a tile
 * with more than 1024 such keys sends its row the long way: four digit
 * rounds over the row, then a selection in index order).  Rows of at most
 * 2^17 elements with 256 < k <= 8192: one round of 8-bit digit counts finds
 * the key byte of each row's k-th largest, the keys at or above it are
 * gathered and one workgroup per row sorts them (at most 16384 per row; a
 * row with more is finished by its workgroup with three more rounds over
 * the row).  Other shapes: four rounds of digit counts find the k-th key,
 * one stable split keeps the top k in index order, and a row sort orders
 * them.  scratch as in topp_sample_f32, of libscan_scratch_bytes(
 * LIBSCAN_OP_TOPK, rows, len, k) bytes (8192 per tile for the first route,
 * 8 * min(len, 16384) per row for the second, 16 per kept element for the
 * third).  No output may overlap an input or the other output.  Workspace:
 * LIBSCAN_OP_TOPK with (n = k, rows, len). */
int topk_rows_f32(const float* x, float* values_out, int32_t* idx_out, int64_t rows, int64_t len,
                  int64_t k, int largest, void* scratch, size_t scratch_bytes, void* ws,
                  size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the
 * inclusive int32 scan of scan_inclusive_i32, same result, same kernels,
 * but without a workspace argument.  Its workspace is a 4 MiB + 256 B array
 * in the library's own device memory, one per GPU, set up by the first call
 * on each device (its address looked up, then zero-filled by a kernel on
 * `stream`, so make that first call outside graph capture or accept that a
 * captured graph re-zeroes it on every replay) and held until the process
 * ends.  The call itself allocates nothing (no hipMalloc, no library
 * allocation).  n <= LIBSCAN_NOALLOC_MAX_N (2^31) elements, else
 * LIBSCAN_ERANGE; other argument checks as scan_inclusive_i32 (x == y
 * allowed); LIBSCAN_EHIP if the array cannot be set up.  x, y and stream
 * must belong to the current device.  Every call on one GPU shares that
 * GPU's array: calls that may overlap on one GPU (different streams, other
 * threads) race and give wrong results; serialise them, or use the
 * workspace entry points.
 * ------------------------------------------------------------------------ */
#define LIBSCAN_NOALLOC_MAX_N (INT64_C(1) << 31)
int scan_inclusive_i32_noalloc(const int32_t* x, int32_t* y, int64_t n, void* stream);

/* Scratch bytes (see topp_sample_f32) that op needs for rows x len (k: the
 * top-k count, else ignored).  Writes *bytes and returns LIBSCAN_OK, or
 * LIBSCAN_EINVAL for an op without scratch / negative size / NULL bytes,
 * LIBSCAN_ERANGE beyond the op's limits.  Pure host function. */
int libscan_scratch_bytes(int op, int64_t rows, int64_t len, int64_t k, size_t* bytes);

#ifdef __cplusplus
}
#endif

#endif /* LIBSCAN_H */
