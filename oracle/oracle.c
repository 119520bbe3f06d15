/*
 * oracle.c -- serial CPU reference for the scan hot path.
 *
 * TEST INFRASTRUCTURE ONLY: used by the tests, the smoke check and the
 * benchmark's CPU-baseline leg, never by the product path.  It shares no code
 * with the HIP library.
 *
 * Every function below is the plain definition of the operation named in its
 * comment (sections of "Parallel Scan on Ascend AI Accelerators"), written as
 * one serial loop in index order.  Integer sums wrap modulo 2^32 because they
 * are accumulated in uint32_t; floating-point sums are accumulated in double.
 */
#include "oracle.h"

#include <math.h>
#include <string.h>
#include <stdlib.h>

/* ---- Section 2: inclusive prefix sum, y_i = x_1 + x_2 + ... + x_i -------- */

void oracle_scan_inclusive_i32(const int32_t* x, uint32_t* y, int64_t n) {
    uint32_t acc = 0;
    for (int64_t i = 0; i < n; ++i) {
        acc += (uint32_t)x[i];
        y[i] = acc;
    }
}

/* ---- Appendix "Exclusive and int8 scan": zero first, then the inclusive
 *      sums shifted by one place, the last one dropped --------------------- */

void oracle_scan_exclusive_i32(const int32_t* x, uint32_t* y, int64_t n) {
    uint32_t acc = 0;
    for (int64_t i = 0; i < n; ++i) {
        y[i] = acc;
        acc += (uint32_t)x[i];
    }
}

void oracle_scan_inclusive_f32(const float* x, double* y, double* a, int64_t n) {
    double acc = 0.0, aacc = 0.0;
    for (int64_t i = 0; i < n; ++i) {
        acc += (double)x[i];
        aacc += fabs((double)x[i]);
        y[i] = acc;
        if (a) a[i] = aacc;
    }
}

void oracle_scan_exclusive_f32(const float* x, double* y, double* a, int64_t n) {
    double acc = 0.0, aacc = 0.0;
    for (int64_t i = 0; i < n; ++i) {
        y[i] = acc;
        if (a) a[i] = aacc;
        acc += (double)x[i];
        aacc += fabs((double)x[i]);
    }
}

/* IEEE 754-2008 binary16: 1 sign bit, 5 exponent bits (bias 15), 10 fraction
 * bits.  Exponent field 0 encodes zero and the subnormals f * 2^-24; field 31
 * encodes infinity (f = 0) and NaN (f != 0); any other field e encodes
 * (1024 + f) * 2^(e - 25).  Every binary16 value is exact in double. */
double oracle_half_to_double(uint16_t h) {
    const int sign = (h >> 15) & 1;
    const int e = (h >> 10) & 31;
    const int f = h & 1023;
    double v;
    if (e == 0) {
        v = ldexp((double)f, -24);
    } else if (e == 31) {
        v = (f == 0) ? INFINITY : NAN;
    } else {
        v = ldexp((double)(1024 + f), e - 25);
    }
    return sign ? -v : v;
}

void oracle_scan_inclusive_f16(const uint16_t* x, double* y, double* a, int64_t n) {
    double acc = 0.0, aacc = 0.0;
    for (int64_t i = 0; i < n; ++i) {
        const double v = oracle_half_to_double(x[i]);
        acc += v;
        aacc += fabs(v);
        y[i] = acc;
        if (a) a[i] = aacc;
    }
}

void oracle_scan_exclusive_f16(const uint16_t* x, double* y, double* a, int64_t n) {
    double acc = 0.0, aacc = 0.0;
    for (int64_t i = 0; i < n; ++i) {
        const double v = oracle_half_to_double(x[i]);
        y[i] = acc;
        if (a) a[i] = aacc;
        acc += v;
        aacc += fabs(v);
    }
}

void oracle_scan_exclusive_u8(const uint8_t* x, uint32_t* y, int64_t n, uint32_t* total) {
    uint32_t acc = 0;
    for (int64_t i = 0; i < n; ++i) {
        y[i] = acc;
        acc += (uint32_t)x[i];
    }
    if (total) *total = acc;
}

void oracle_scan_inclusive_u8(const uint8_t* x, uint32_t* y, int64_t n) {
    uint32_t acc = 0;
    for (int64_t i = 0; i < n; ++i) {
        acc += (uint32_t)x[i];
        y[i] = acc;
    }
}

/* ---- Appendix "Multiple (Batched) Scans": every row on its own ---------- */

void oracle_scan_rows_i32(const int32_t* x, uint32_t* y, int64_t rows, int64_t len,
                          int exclusive) {
    for (int64_t r = 0; r < rows; ++r) {
        if (exclusive)
            oracle_scan_exclusive_i32(x + r * len, y + r * len, len);
        else
            oracle_scan_inclusive_i32(x + r * len, y + r * len, len);
    }
}

void oracle_scan_rows_f32(const float* x, double* y, double* a, int64_t rows, int64_t len,
                          int exclusive) {
    for (int64_t r = 0; r < rows; ++r) {
        double* ar = a ? a + r * len : 0;
        if (exclusive)
            oracle_scan_exclusive_f32(x + r * len, y + r * len, ar, len);
        else
            oracle_scan_inclusive_f32(x + r * len, y + r * len, ar, len);
    }
}

/* ---- Section 5 "Compress": torch.masked_select order -------------------- */

int64_t oracle_compact_f32(const float* x, const uint8_t* mask, float* out, int32_t* idx,
                           int64_t n) {
    int64_t c = 0;
    for (int64_t i = 0; i < n; ++i) {
        if (mask[i] != 0) {
            out[c] = x[i];
            if (idx) idx[c] = (int32_t)i;
            ++c;
        }
    }
    return c;
}

/* ---- Section 5 "Split": flagged items first, then the rest, both stable -- */

int64_t oracle_split_u32(const uint32_t* keys, const int32_t* idx_in, const uint8_t* flags,
                         uint32_t* keys_out, int32_t* idx_out, int64_t n) {
    int64_t c = 0;
    for (int64_t i = 0; i < n; ++i) { /* first pass: the flagged items */
        if (flags[i] != 0) {
            keys_out[c] = keys[i];
            if (idx_out) idx_out[c] = idx_in ? idx_in[i] : (int32_t)i;
            ++c;
        }
    }
    const int64_t n_true = c;
    for (int64_t i = 0; i < n; ++i) { /* second pass: the unflagged items */
        if (flags[i] == 0) {
            keys_out[c] = keys[i];
            if (idx_out) idx_out[c] = idx_in ? idx_in[i] : (int32_t)i;
            ++c;
        }
    }
    return n_true;
}

/* ---- Section 5 "Radix Sort": the stable ascending order it must produce - */

typedef struct {
    uint32_t key;
    int32_t index;
} oracle_pair;

static int oracle_pair_less(const void* pa, const void* pb) {
    const oracle_pair* a = (const oracle_pair*)pa;
    const oracle_pair* b = (const oracle_pair*)pb;
    if (a->key != b->key) return a->key < b->key ? -1 : 1;
    return a->index < b->index ? -1 : (a->index > b->index ? 1 : 0);
}

int oracle_sort_u32(const uint32_t* keys, uint32_t* keys_out, int32_t* perm_out, int64_t n) {
    if (n <= 0) return 0;
    oracle_pair* p = (oracle_pair*)malloc((size_t)n * sizeof(oracle_pair));
    if (!p) return -1;
    for (int64_t i = 0; i < n; ++i) {
        p[i].key = keys[i];
        p[i].index = (int32_t)i;
    }
    /* (key, index) pairs are all distinct, so their order is total and the
     * result is unique even though qsort itself is not stable. */
    qsort(p, (size_t)n, sizeof(oracle_pair), oracle_pair_less);
    for (int64_t i = 0; i < n; ++i) {
        keys_out[i] = p[i].key;
        perm_out[i] = p[i].index;
    }
    free(p);
    return 0;
}

/* ---- Section 5 "Radix Sort" on signed and floating-point keys ---------- */

/* Order of two keys of one type: -1, 0 or 1.  Floats follow IEEE 754
 * totalOrder, written from its definition: numbers by value, the two zeros by
 * sign, NaNs outside everything by sign and among themselves by payload. */
static int oracle_cmp_i32(uint64_t a, uint64_t b) {
    const int32_t x = (int32_t)(uint32_t)a, y = (int32_t)(uint32_t)b;
    return x < y ? -1 : (x > y ? 1 : 0);
}

static int oracle_cmp_float(double x, double y, int sx, int sy, int nanx, int nany, uint32_t payx,
                            uint32_t payy) {
    if (!nanx && !nany) {
        if (x < y) return -1;
        if (x > y) return 1;
        if (sx != sy) return sx ? -1 : 1; /* -0 before +0 */
        return 0;
    }
    if (nanx && nany) {
        if (sx != sy) return sx ? -1 : 1;
        if (payx == payy) return 0;
        /* larger payload farther from zero: later if positive, earlier if negative */
        return ((payx < payy) != (sx != 0)) ? -1 : 1;
    }
    if (nanx) return sx ? -1 : 1;
    return sy ? 1 : -1;
}

static int oracle_cmp_f32(uint64_t a, uint64_t b) {
    float x, y;
    const uint32_t ba = (uint32_t)a, bb = (uint32_t)b;
    memcpy(&x, &ba, 4);
    memcpy(&y, &bb, 4);
    return oracle_cmp_float(x, y, (int)(ba >> 31), (int)(bb >> 31), isnan(x), isnan(y),
                            ba & 0x7fffffu, bb & 0x7fffffu);
}

static int oracle_cmp_f16(uint64_t a, uint64_t b) {
    const uint16_t ha = (uint16_t)a, hb = (uint16_t)b;
    const double x = oracle_half_to_double(ha), y = oracle_half_to_double(hb);
    return oracle_cmp_float(x, y, ha >> 15, hb >> 15, isnan(x), isnan(y), ha & 0x3ffu,
                            hb & 0x3ffu);
}

typedef struct {
    uint64_t key;
    int32_t index;
} oracle_kpair;

/* qsort comparators take no context: the key order and direction are set
 * here for the duration of one call (the oracle is single-threaded). */
static int (*oracle_kcmp)(uint64_t, uint64_t);
static int oracle_kdesc;

static int oracle_kpair_less(const void* pa, const void* pb) {
    const oracle_kpair* a = (const oracle_kpair*)pa;
    const oracle_kpair* b = (const oracle_kpair*)pb;
    int c = oracle_kcmp(a->key, b->key);
    if (oracle_kdesc) c = -c;
    if (c != 0) return c;
    return (a->index > b->index) - (a->index < b->index); /* ties: index order */
}

static int oracle_sort_keys(const void* keys, void* keys_out, int32_t* perm_out, int64_t n,
                            int bytes, int (*cmp)(uint64_t, uint64_t), int descending) {
    if (n <= 0) return 0;
    oracle_kpair* p = (oracle_kpair*)malloc((size_t)n * sizeof(oracle_kpair));
    if (!p) return -1;
    for (int64_t i = 0; i < n; ++i) {
        p[i].key = bytes == 4 ? ((const uint32_t*)keys)[i] : ((const uint16_t*)keys)[i];
        p[i].index = (int32_t)i;
    }
    oracle_kcmp = cmp;
    oracle_kdesc = descending != 0;
    qsort(p, (size_t)n, sizeof(oracle_kpair), oracle_kpair_less);
    for (int64_t i = 0; i < n; ++i) {
        if (bytes == 4)
            ((uint32_t*)keys_out)[i] = (uint32_t)p[i].key;
        else
            ((uint16_t*)keys_out)[i] = (uint16_t)p[i].key;
        perm_out[i] = p[i].index;
    }
    free(p);
    return 0;
}

int oracle_sort_i32(const int32_t* keys, int32_t* keys_out, int32_t* perm_out, int64_t n,
                    int descending) {
    return oracle_sort_keys(keys, keys_out, perm_out, n, 4, oracle_cmp_i32, descending);
}

int oracle_sort_f32(const uint32_t* keys, uint32_t* keys_out, int32_t* perm_out, int64_t n,
                    int descending) {
    return oracle_sort_keys(keys, keys_out, perm_out, n, 4, oracle_cmp_f32, descending);
}

int oracle_sort_f16(const uint16_t* keys, uint16_t* keys_out, int32_t* perm_out, int64_t n,
                    int descending) {
    return oracle_sort_keys(keys, keys_out, perm_out, n, 2, oracle_cmp_f16, descending);
}

/* ---- Section 5 "Top-p": first index whose running probability mass
 *      reaches p, keeping every token up to and including it ------------- */

void oracle_topp_cutoff_f32(const float* probs, int32_t* cutoff, int64_t rows, int64_t len,
                            float p) {
    const double pd = (double)p;
    for (int64_t r = 0; r < rows; ++r) {
        const float* row = probs + r * len;
        double c = 0.0;
        int64_t k = len - 1;
        for (int64_t i = 0; i < len; ++i) {
            c += (double)row[i];
            if (c >= pd) {
                k = i;
                break;
            }
        }
        cutoff[r] = (int32_t)k;
    }
}

/* ---- Batched sorts and the samplers ------------------------------------ */

int oracle_sort_rows_f32(const uint32_t* keys, uint32_t* keys_out, int32_t* idx_out, int64_t rows,
                         int64_t len, int descending) {
    for (int64_t r = 0; r < rows; ++r)
        if (oracle_sort_f32(keys + r * len, keys_out + r * len, idx_out + r * len, len,
                            descending) != 0)
            return -1;
    return 0;
}

int oracle_topk_rows_f32(const uint32_t* x, uint32_t* values_out, int32_t* idx_out, int64_t rows,
                         int64_t len, int64_t k, int largest) {
    if (k < 0 || k > len) return -1;
    if (len == 0 || k == 0) return 0;
    uint32_t* sorted = (uint32_t*)malloc((size_t)len * sizeof(uint32_t));
    int32_t* idx = (int32_t*)malloc((size_t)len * sizeof(int32_t));
    int rc = (sorted && idx) ? 0 : -1;
    for (int64_t r = 0; r < rows && rc == 0; ++r) {
        rc = oracle_sort_f32(x + r * len, sorted, idx, len, largest != 0);
        for (int64_t i = 0; i < k && rc == 0; ++i) {
            values_out[r * k + i] = sorted[i];
            idx_out[r * k + i] = idx[i];
        }
    }
    free(sorted);
    free(idx);
    return rc;
}

/* First i in [0, limit] with s[i] > u (running sums in double), else limit. */
static int64_t oracle_first_above(const float* w, int64_t limit, double u) {
    double acc = 0.0;
    for (int64_t i = 0; i <= limit; ++i) {
        acc += (double)w[i];
        if (acc > u) return i;
    }
    return limit;
}

void oracle_weighted_sample_f32(const float* w, const float* theta, int32_t* out, int64_t rows,
                                int64_t len) {
    for (int64_t r = 0; r < rows; ++r) {
        const float* row = w + r * len;
        if (len == 0) {
            out[r] = -1;
            continue;
        }
        double total = 0.0;
        for (int64_t i = 0; i < len; ++i) total += (double)row[i];
        out[r] = (int32_t)oracle_first_above(row, len - 1, (double)theta[r] * total);
    }
}

int oracle_topp_sample_f32(const float* probs, const float* theta, float p, int32_t* token_out,
                           int32_t* cutoff_out, int64_t rows, int64_t len) {
    if (len == 0) {
        for (int64_t r = 0; r < rows; ++r) {
            token_out[r] = -1;
            if (cutoff_out) cutoff_out[r] = -1;
        }
        return 0;
    }
    uint32_t* sorted = (uint32_t*)malloc((size_t)len * sizeof(uint32_t));
    int32_t* idx = (int32_t*)malloc((size_t)len * sizeof(int32_t));
    if (!sorted || !idx) {
        free(sorted);
        free(idx);
        return -1;
    }
    int rc = 0;
    for (int64_t r = 0; r < rows && rc == 0; ++r) {
        rc = oracle_sort_f32((const uint32_t*)(probs + r * len), sorted, idx, len, 1);
        if (rc != 0) break;
        const float* s = (const float*)sorted;
        int32_t k;
        oracle_topp_cutoff_f32(s, &k, 1, len, p);
        double ck = 0.0;
        for (int64_t i = 0; i <= k; ++i) ck += (double)s[i];
        const int64_t j = oracle_first_above(s, k, (double)theta[r] * ck);
        token_out[r] = idx[j];
        if (cutoff_out) cutoff_out[r] = k;
    }
    free(sorted);
    free(idx);
    return rc;
}
