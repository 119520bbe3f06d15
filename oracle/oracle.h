/*
 * oracle.h -- serial CPU reference for the scan hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path (the HIP library and
 * its Python binding) includes, links or calls this code.  Only the tests, the
 * smoke check and the benchmark's CPU-baseline leg use it.
 *
 * Each function is the plain definition of what an operation of
 * "Parallel Scan on Ascend AI Accelerators" (Wroblewski, Gottardo, Zouzias)
 * computes, written as one serial loop: no tiling, no reordering.
 *   - integer sums wrap modulo 2^32 (accumulated in uint32_t);
 *   - floating-point sums are accumulated in double and returned in double,
 *     together with the running sum of |x| that the float tolerance uses.
 * All pointers are host pointers owned by the caller; nothing is allocated
 * except the temporary arrays of the sorts.
 */
#ifndef LIBSCAN_ORACLE_H
#define LIBSCAN_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Section 2 (Background): the inclusive prefix sum y_i = x_1 + ... + x_i. */
void oracle_scan_inclusive_i32(const int32_t* x, uint32_t* y, int64_t n);
/* Appendix "Exclusive and int8 scan": the inclusive result shifted right by
 * one, the last value dropped, zero in front. */
void oracle_scan_exclusive_i32(const int32_t* x, uint32_t* y, int64_t n);

/* Float scans: y = prefix sums in double, a = prefix sums of |x| in double
 * (a may be NULL). */
void oracle_scan_inclusive_f32(const float* x, double* y, double* a, int64_t n);
void oracle_scan_exclusive_f32(const float* x, double* y, double* a, int64_t n);

/* IEEE 754 binary16 bit pattern -> exact double value. */
double oracle_half_to_double(uint16_t h);
/* fp16 input (raw bit patterns), every value converted exactly to double. */
void oracle_scan_inclusive_f16(const uint16_t* x, double* y, double* a, int64_t n);
void oracle_scan_exclusive_f16(const uint16_t* x, double* y, double* a, int64_t n);

/* Appendix "Exclusive and int8 scan": 8-bit inputs summed as integers into a
 * 32-bit result (mod 2^32).  *total (may be NULL) receives the full sum. */
void oracle_scan_exclusive_u8(const uint8_t* x, uint32_t* y, int64_t n, uint32_t* total);
void oracle_scan_inclusive_u8(const uint8_t* x, uint32_t* y, int64_t n);

/* Appendix "Multiple (Batched) Scans": an independent scan of every row of a
 * row-major rows x len matrix. */
void oracle_scan_rows_i32(const int32_t* x, uint32_t* y, int64_t rows, int64_t len, int exclusive);
void oracle_scan_rows_f32(const float* x, double* y, double* a, int64_t rows, int64_t len,
                          int exclusive);

/* Section 5 "Compress": keep x_i where mask_i != 0, in index order; idx (may
 * be NULL) receives the source indices.  Returns the number kept. */
int64_t oracle_compact_f32(const float* x, const uint8_t* mask, float* out, int32_t* idx,
                           int64_t n);

/* Section 5 "Split": the flagged items first, then the unflagged ones, each
 * group in index order.  idx_in NULL means the identity.  Returns the number
 * flagged. */
int64_t oracle_split_u32(const uint32_t* keys, const int32_t* idx_in, const uint8_t* flags,
                         uint32_t* keys_out, int32_t* idx_out, int64_t n);

/* Section 5 "Radix Sort": the result radix sort must reach -- a stable
 * ascending sort of unsigned keys.  perm_out[i] is the source index of
 * keys_out[i].  Defined as the lexicographic order of (key, source index).
 * Returns 0, or -1 if the temporary array cannot be allocated. */
int oracle_sort_u32(const uint32_t* keys, uint32_t* keys_out, int32_t* perm_out, int64_t n);

/* Section 5 "Radix Sort" on signed integer and floating-point keys (the
 * paper sorts fp16 and supports signed integers and floats): a stable sort,
 * ascending or (descending != 0) descending, ties kept in index order.
 * Integers compare as integers.  Floats compare in IEEE 754 totalOrder:
 * numerical order, -0 before +0, NaNs with the sign bit set below everything
 * and the others above, NaNs of one sign ordered by payload (larger payload
 * farther from zero).  Keys are copied as bit patterns.  Return 0, or -1 if
 * the temporary array cannot be allocated. */
int oracle_sort_i32(const int32_t* keys, int32_t* keys_out, int32_t* perm_out, int64_t n,
                    int descending);
int oracle_sort_f32(const uint32_t* keys, uint32_t* keys_out, int32_t* perm_out, int64_t n,
                    int descending);
int oracle_sort_f16(const uint16_t* keys, uint16_t* keys_out, int32_t* perm_out, int64_t n,
                    int descending);

/* Batched form of the float sort (as the appendix "Multiple (Batched) Scans"
 * batches scans): every row of a row-major rows x len matrix sorted on its own,
 * stably; idx_out holds each key's index within its row. */
int oracle_sort_rows_f32(const uint32_t* keys, uint32_t* keys_out, int32_t* idx_out, int64_t rows,
                         int64_t len, int descending);

/* Section 5 "Top-k": per row, the k largest (largest != 0) or the k smallest
 * values in IEEE 754 totalOrder, listed in that order (descending or
 * ascending), equal values by increasing index: the first k entries of the
 * row's stable sort in that direction.  values_out (bit copies) and idx_out
 * (indices within the row) are rows x k.  0 <= k <= len.  Returns 0, or -1 on
 * allocation failure. */
int oracle_topk_rows_f32(const uint32_t* x, uint32_t* values_out, int32_t* idx_out, int64_t rows,
                         int64_t len, int64_t k, int largest);

/* Appendix "Weighted Sampling": inverse transform sampling from the scan of
 * the weights.  Per row, with S_i the inclusive running sum (in double) and
 * W = S_{len-1}: the first index with S_i > theta * W (len - 1 if rounding
 * leaves none; -1 for len = 0). */
void oracle_weighted_sample_f32(const float* w, const float* theta, int32_t* out, int64_t rows,
                                int64_t len);

/* Section 5 "Top-p or Nucleus Sampling" as a whole sampler: per row of
 * (unsorted) probabilities, sort them in descending order (stably), take the
 * cutoff k of the sorted row (oracle_topp_cutoff_f32), and draw one of the
 * kept tokens 0..k by inverse transform: the first i <= k whose running sum
 * exceeds theta * C_k (k if rounding leaves none).  token_out is the drawn
 * token's index in the unsorted row; cutoff_out (nullable) receives k.
 * len = 0 gives -1 for both.  Returns 0, or -1 on allocation failure. */
int oracle_topp_sample_f32(const float* probs, const float* theta, float p, int32_t* token_out,
                           int32_t* cutoff_out, int64_t rows, int64_t len);

/* Section 5 "Top-p or Nucleus Sampling": per row of probabilities already
 * sorted in descending order, the first index whose inclusive running sum
 * (in double) reaches p, or len - 1 if it never does. */
void oracle_topp_cutoff_f32(const float* probs, int32_t* cutoff, int64_t rows, int64_t len,
                            float p);

#ifdef __cplusplus
}
#endif

#endif
