// abi.hip -- the extern "C" entry points of libscan (declared in libscan.h).
//
// Each entry point checks its arguments on the host, before any HIP call, and
// then enqueues the kernels through the launchers of launch.hpp.
#include <limits.h>
#include <string.h>

#include "../../include/libscan.h"
#include "launch.hpp"

namespace {

using ls::Kind;

bool overlaps(const void* a, size_t abytes, const void* b, size_t bbytes) {
    const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
    return abytes && bbytes && a0 < b0 + bbytes && b0 < a0 + abytes;
}

// Output [y, y+ybytes) against input [x, x+xbytes): exact aliasing is fine
// when `inplace_ok` (same start, same size), any other overlap is not.
bool bad_alias(const void* x, size_t xbytes, const void* y, size_t ybytes, bool inplace_ok) {
    if (!overlaps(x, xbytes, y, ybytes)) return false;
    return !(inplace_ok && x == y && xbytes == ybytes);
}

int hip_status(hipError_t e) { return e == hipSuccess ? LIBSCAN_OK : LIBSCAN_EHIP; }

int check_ws(void* ws, size_t ws_bytes, size_t need) {
    if (ws_bytes < need) return LIBSCAN_ENOSPACE;
    if (!ws || ((uintptr_t)ws % 16) != 0) return LIBSCAN_EINVAL;
    return LIBSCAN_OK;
}

size_t elem_bytes_in(Kind k) {
    switch (k) {
        case Kind::I32:
        case Kind::F32:
            return 4;
        case Kind::F16F32:
            return 2;
        case Kind::U8I32:
            return 1;
    }
    return 0;
}

int scan1d(Kind kind, bool exclusive, const void* x, void* y, int64_t n, const void* carry_in,
           void* total_out, void* ws, size_t ws_bytes, void* stream) {
    if (n < 0) return LIBSCAN_EINVAL;
    if (n > ls::kMaxScanElems) return LIBSCAN_ERANGE;
    if (n > 0 && (!x || !y)) return LIBSCAN_EINVAL;
    const size_t in_b = (size_t)n * elem_bytes_in(kind), out_b = (size_t)n * 4;
    const bool same_type = kind == Kind::I32 || kind == Kind::F32;
    if (bad_alias(x, in_b, y, out_b, same_type)) return LIBSCAN_EINVAL;
    if (total_out && overlaps(total_out, 4, y, out_b)) return LIBSCAN_EINVAL;
    if (n == 0 && !total_out) return LIBSCAN_OK;
    const int w = check_ws(ws, ws_bytes, ls::scan1d_ws_bytes(n));
    if (w != LIBSCAN_OK) return w;
    return hip_status(ls::launch_scan1d(kind, exclusive, x, y, n, carry_in, total_out, ws,
                                        ws_bytes, (hipStream_t)stream));
}

int scan1d_rss(Kind kind, const void* x, void* y, int64_t n, void* ws, size_t ws_bytes,
               void* stream) {
    if (n < 0) return LIBSCAN_EINVAL;
    if (n > ls::kMaxScanElems) return LIBSCAN_ERANGE;
    if (n > 0 && (!x || !y)) return LIBSCAN_EINVAL;
    if (bad_alias(x, (size_t)n * 4, y, (size_t)n * 4, true)) return LIBSCAN_EINVAL;
    if (n == 0) return LIBSCAN_OK;
    const int w = check_ws(ws, ws_bytes, ls::scan1d_rss_ws_bytes(n));
    if (w != LIBSCAN_OK) return w;
    return hip_status(ls::launch_scan1d_rss(kind, x, y, n, ws, (hipStream_t)stream));
}

// rows x len must describe at most kMaxScanElems elements and a tile grid
// that fits one launch.
int check_rows(int64_t rows, int64_t len) {
    if (rows < 0 || len < 0) return LIBSCAN_EINVAL;
    if (rows > 0 && len > ls::kMaxScanElems / rows) return LIBSCAN_ERANGE;
    if (rows > 0 && len > 0 && rows * ((len + 4095) / 4096) > ls::kMaxGridTiles) return LIBSCAN_ERANGE;
    return LIBSCAN_OK;
}

int scan_rows(Kind kind, const void* x, void* y, int64_t rows, int64_t len, int exclusive,
              void* ws, size_t ws_bytes, void* stream) {
    const int r = check_rows(rows, len);
    if (r != LIBSCAN_OK) return r;
    const size_t bytes = (size_t)rows * (size_t)len * 4;
    if (bytes > 0 && (!x || !y)) return LIBSCAN_EINVAL;
    if (bad_alias(x, bytes, y, bytes, true)) return LIBSCAN_EINVAL;
    if (bytes == 0) return LIBSCAN_OK;
    const int w = check_ws(ws, ws_bytes, ls::scan_rows_ws_bytes(rows, len));
    if (w != LIBSCAN_OK) return w;
    return hip_status(ls::launch_scan_rows(kind, exclusive != 0, x, y, rows, len, ws, ws_bytes,
                                           (hipStream_t)stream));
}

int radix_sort_typed(ls::KeyType type, size_t elem, const void* keys, void* keys_out,
                     int32_t* perm_out, void* keys_tmp, int32_t* perm_tmp, int64_t n,
                     int descending, void* ws, size_t ws_bytes, void* stream) {
    if (n < 0) return LIBSCAN_EINVAL;
    if (n > ls::kMaxRadixKeys) return LIBSCAN_ERANGE;
    if (n == 0) return LIBSCAN_OK;
    if (!keys || !keys_out || !keys_tmp || (perm_out && !perm_tmp)) return LIBSCAN_EINVAL;
    const size_t kb = (size_t)n * elem, pb = (size_t)n * 4;
    const void* bufs[5] = {keys, keys_out, perm_out, keys_tmp, perm_out ? perm_tmp : nullptr};
    const size_t len[5] = {kb, kb, perm_out ? pb : 0, kb, perm_out ? pb : 0};
    for (int i = 0; i < 5; ++i)
        for (int j = i + 1; j < 5; ++j)
            if (overlaps(bufs[i], bufs[i] ? len[i] : 0, bufs[j], bufs[j] ? len[j] : 0))
                return LIBSCAN_EINVAL;
    const int w = check_ws(ws, ws_bytes, ls::radix_ws_bytes(n, 8));
    if (w != LIBSCAN_OK) return w;
    return hip_status(ls::launch_radix_sort_typed(type, descending != 0, keys, keys_out, nullptr,
                                                  perm_out, keys_tmp, perm_tmp, 1, n, ws, ws_bytes,
                                                  (hipStream_t)stream));
}

// Per-row sampling ops: rows x len probabilities or weights in, one int32
// per row out, theta (rows floats) read by the draw.
int check_sample(const float* x, const float* theta, const int32_t* out, const int32_t* out2,
                 int64_t rows, int64_t len) {
    const int r = check_rows(rows, len);
    if (r != LIBSCAN_OK) return r;
    if (len > INT32_MAX) return LIBSCAN_ERANGE;
    if (rows == 0) return LIBSCAN_OK;
    if (!theta || !out || (len > 0 && !x)) return LIBSCAN_EINVAL;
    const size_t xb = (size_t)rows * (size_t)len * 4, rb = (size_t)rows * 4;
    if (overlaps(out, rb, x, xb) || overlaps(out, rb, theta, rb) ||
        overlaps(out2, out2 ? rb : 0, x, xb) || overlaps(out2, out2 ? rb : 0, theta, rb) ||
        overlaps(out2, out2 ? rb : 0, out, rb))
        return LIBSCAN_EINVAL;
    return LIBSCAN_OK;
}

// Top-k sizes: 0 <= k <= len, the row grid as scan_rows, the k kept per row
// as a row sort.
int check_topk(int64_t rows, int64_t len, int64_t k) {
    if (rows < 0 || len < 0 || k < 0 || k > len) return LIBSCAN_EINVAL;
    const int r = check_rows(rows, len);
    if (r != LIBSCAN_OK) return r;
    if (len > INT32_MAX || !ls::radix_rows_fit(rows, k)) return LIBSCAN_ERANGE;
    return LIBSCAN_OK;
}

int scan_u8_variant(bool mfma, const uint8_t* x, int32_t* y, int64_t n, int32_t* total_dev,
                           void* ws, size_t ws_bytes, void* stream) {
    if (n < 0) return LIBSCAN_EINVAL;
    if (n > ls::kMaxScanElems) return LIBSCAN_ERANGE;
    if (n > 0 && (!x || !y)) return LIBSCAN_EINVAL;
    if (bad_alias(x, (size_t)n, y, (size_t)n * 4, false)) return LIBSCAN_EINVAL;
    if (total_dev && overlaps(total_dev, 4, y, (size_t)n * 4)) return LIBSCAN_EINVAL;
    if (n == 0 && !total_dev) return LIBSCAN_OK;
    if (mfma && n > 0 && (((uintptr_t)x % 16) != 0 || ((uintptr_t)y % 4) != 0))
        return LIBSCAN_EINVAL;
    const int w = check_ws(ws, ws_bytes, ls::scan1d_ws_bytes(n));
    if (w != LIBSCAN_OK) return w;
    hipStream_t s = (hipStream_t)stream;
    if (mfma && n > 0)
        return hip_status(ls::launch_scan1d_mfma_u8(x, (uint32_t*)y, n, (uint32_t*)total_dev, ws,
                                                    ws_bytes, s));
    return hip_status(ls::launch_scan1d_tiles(Kind::U8I32, true, x, y, n, nullptr, total_dev, ws,
                                              ws_bytes, s));
}

}  // namespace

extern "C" {

int libscan_version(void) { return 100; }

const char* libscan_status_string(int status) {
    switch (status) {
        case LIBSCAN_OK:
            return "success";
        case LIBSCAN_EINVAL:
            return "invalid argument";
        case LIBSCAN_ENOSPACE:
            return "workspace too small";
        case LIBSCAN_EHIP:
            return "HIP launch error";
        case LIBSCAN_ERANGE:
            return "size out of range";
        default:
            return "unknown status";
    }
}

int libscan_workspace_init(void* ws, size_t ws_bytes, void* stream) {
    if (ws_bytes == 0) return LIBSCAN_OK;
    if (!ws || ((uintptr_t)ws % 16) != 0 || ws_bytes % 8 != 0) return LIBSCAN_EINVAL;
    return hip_status(ls::launch_workspace_init(ws, ws_bytes, (hipStream_t)stream));
}

int libscan_workspace_error(void* ws, size_t ws_bytes, int32_t* error_dev, int reset,
                            void* stream) {
    if (!ws || ((uintptr_t)ws % 16) != 0 || !error_dev || ((uintptr_t)error_dev % 4) != 0)
        return LIBSCAN_EINVAL;
    if (ws_bytes < ls::kWsHeader) return LIBSCAN_ENOSPACE;
    if (overlaps(error_dev, 4, ws, ls::kWsHeader)) return LIBSCAN_EINVAL;
    return hip_status(ls::launch_workspace_error(ws, error_dev, reset != 0, (hipStream_t)stream));
}

int libscan_workspace_bytes(int op, int64_t n, int64_t rows, int64_t len, int bits, size_t* bytes) {
    if (!bytes || n < 0 || rows < 0 || len < 0) return LIBSCAN_EINVAL;
    switch (op) {
        case LIBSCAN_OP_SCAN:
            if (n > ls::kMaxScanElems) return LIBSCAN_ERANGE;
            *bytes = ls::scan1d_ws_bytes(n);
            return LIBSCAN_OK;
        case LIBSCAN_OP_SCAN_RSS:
            if (n > ls::kMaxScanElems) return LIBSCAN_ERANGE;
            *bytes = ls::scan1d_rss_ws_bytes(n);
            return LIBSCAN_OK;
        case LIBSCAN_OP_COMPACT:
            if (n > INT32_MAX) return LIBSCAN_ERANGE;
            *bytes = ls::compact_ws_bytes(n);
            return LIBSCAN_OK;
        case LIBSCAN_OP_RADIX_SORT:
            if (n > ls::kMaxRadixKeys) return LIBSCAN_ERANGE;
            if (bits != 1 && bits != 4 && bits != 8) return LIBSCAN_EINVAL;
            *bytes = ls::radix_ws_bytes(n, bits);
            return LIBSCAN_OK;
        case LIBSCAN_OP_SCAN_ROWS: {
            const int r = check_rows(rows, len);
            if (r != LIBSCAN_OK) return r;
            *bytes = ls::scan_rows_ws_bytes(rows, len);
            return LIBSCAN_OK;
        }
        case LIBSCAN_OP_SORT_ROWS:
            if (!ls::radix_rows_fit(rows, len)) return LIBSCAN_ERANGE;
            *bytes = ls::radix_rows_ws_bytes(rows, len);
            return LIBSCAN_OK;
        case LIBSCAN_OP_TOPK: {
            const int r = check_topk(rows, len, n);
            if (r != LIBSCAN_OK) return r;
            *bytes = ls::topk_ws_bytes(rows, len, n);
            return LIBSCAN_OK;
        }
        case LIBSCAN_OP_WEIGHTED_SAMPLE:
        case LIBSCAN_OP_TOPP_SAMPLE: {
            const int r = check_rows(rows, len);
            if (r != LIBSCAN_OK) return r;
            if (len > INT32_MAX) return LIBSCAN_ERANGE;
            if (op == LIBSCAN_OP_WEIGHTED_SAMPLE) {
                *bytes = ls::weighted_ws_bytes(rows, len);
            } else {
                if (!ls::radix_rows_fit(rows, len)) return LIBSCAN_ERANGE;
                *bytes = ls::topp_sample_ws_bytes(rows, len);
            }
            return LIBSCAN_OK;
        }
        default:
            return LIBSCAN_EINVAL;
    }
}

int scan_inclusive_i32(const int32_t* x, int32_t* y, int64_t n, void* ws, size_t ws_bytes,
                       void* stream) {
    return scan1d(Kind::I32, false, x, y, n, nullptr, nullptr, ws, ws_bytes, stream);
}
int scan_exclusive_i32(const int32_t* x, int32_t* y, int64_t n, void* ws, size_t ws_bytes,
                       void* stream) {
    return scan1d(Kind::I32, true, x, y, n, nullptr, nullptr, ws, ws_bytes, stream);
}
int scan_inclusive_f32(const float* x, float* y, int64_t n, void* ws, size_t ws_bytes,
                       void* stream) {
    return scan1d(Kind::F32, false, x, y, n, nullptr, nullptr, ws, ws_bytes, stream);
}
int scan_exclusive_f32(const float* x, float* y, int64_t n, void* ws, size_t ws_bytes,
                       void* stream) {
    return scan1d(Kind::F32, true, x, y, n, nullptr, nullptr, ws, ws_bytes, stream);
}
int scan_inclusive_f16f32(const uint16_t* x, float* y, int64_t n, void* ws, size_t ws_bytes,
                          void* stream) {
    return scan1d(Kind::F16F32, false, x, y, n, nullptr, nullptr, ws, ws_bytes, stream);
}
int scan_exclusive_f16f32(const uint16_t* x, float* y, int64_t n, void* ws, size_t ws_bytes,
                          void* stream) {
    return scan1d(Kind::F16F32, true, x, y, n, nullptr, nullptr, ws, ws_bytes, stream);
}

int scan_inclusive_f16f32_wave(const uint16_t* x, float* y, int64_t n, void* ws, size_t ws_bytes,
                               void* stream) {
    if (n < 0) return LIBSCAN_EINVAL;
    if (n > ls::kMaxScanElems) return LIBSCAN_ERANGE;
    if (n > 0 && (!x || !y)) return LIBSCAN_EINVAL;
    if (bad_alias(x, (size_t)n * 2, y, (size_t)n * 4, false)) return LIBSCAN_EINVAL;
    if (n == 0) return LIBSCAN_OK;
    const int w = check_ws(ws, ws_bytes, ls::scan1d_ws_bytes(n));
    if (w != LIBSCAN_OK) return w;
    return hip_status(ls::launch_scan1d_tiles(Kind::F16F32, false, x, y, n, nullptr, nullptr, ws,
                                              ws_bytes, (hipStream_t)stream));
}

int scan_inclusive_f16f32_mfma(const uint16_t* x, float* y, int64_t n, void* ws, size_t ws_bytes,
                               void* stream) {
    if (n < 0) return LIBSCAN_EINVAL;
    if (n > ls::kMaxScanElems) return LIBSCAN_ERANGE;
    if (n > 0 && (!x || !y)) return LIBSCAN_EINVAL;
    if (bad_alias(x, (size_t)n * 2, y, (size_t)n * 4, false)) return LIBSCAN_EINVAL;
    if (n == 0) return LIBSCAN_OK;
    if (((uintptr_t)x % 16) != 0 || ((uintptr_t)y % 4) != 0) return LIBSCAN_EINVAL;
    const int w = check_ws(ws, ws_bytes, ls::scan1d_ws_bytes(n));
    if (w != LIBSCAN_OK) return w;
    return hip_status(ls::launch_scan1d_mfma_f16(x, y, n, ws, ws_bytes, (hipStream_t)stream));
}

int scan_exclusive_u8i32_mfma(const uint8_t* x, int32_t* y, int64_t n, int32_t* total_dev,
                              void* ws, size_t ws_bytes, void* stream) {
    return scan_u8_variant(true, x, y, n, total_dev, ws, ws_bytes, stream);
}

int scan_exclusive_u8i32_wave(const uint8_t* x, int32_t* y, int64_t n, int32_t* total_dev,
                              void* ws, size_t ws_bytes, void* stream) {
    return scan_u8_variant(false, x, y, n, total_dev, ws, ws_bytes, stream);
}
int scan_exclusive_u8i32(const uint8_t* x, int32_t* y, int64_t n, int32_t* total_dev, void* ws,
                         size_t ws_bytes, void* stream) {
    return scan1d(Kind::U8I32, true, x, y, n, nullptr, total_dev, ws, ws_bytes, stream);
}
int scan_inclusive_i32_carry(const int32_t* x, int32_t* y, int64_t n, const int32_t* carry_in_dev,
                             int32_t* total_out_dev, void* ws, size_t ws_bytes, void* stream) {
    return scan1d(Kind::I32, false, x, y, n, carry_in_dev, total_out_dev, ws, ws_bytes, stream);
}
int scan_exclusive_i32_carry(const int32_t* x, int32_t* y, int64_t n, const int32_t* carry_in_dev,
                             int32_t* total_out_dev, void* ws, size_t ws_bytes, void* stream) {
    return scan1d(Kind::I32, true, x, y, n, carry_in_dev, total_out_dev, ws, ws_bytes, stream);
}
int scan_inclusive_f32_carry(const float* x, float* y, int64_t n, const float* carry_in_dev,
                             float* total_out_dev, void* ws, size_t ws_bytes, void* stream) {
    return scan1d(Kind::F32, false, x, y, n, carry_in_dev, total_out_dev, ws, ws_bytes, stream);
}
int scan_exclusive_f32_carry(const float* x, float* y, int64_t n, const float* carry_in_dev,
                             float* total_out_dev, void* ws, size_t ws_bytes, void* stream) {
    return scan1d(Kind::F32, true, x, y, n, carry_in_dev, total_out_dev, ws, ws_bytes, stream);
}
int scan_inclusive_rss_i32(const int32_t* x, int32_t* y, int64_t n, void* ws, size_t ws_bytes,
                           void* stream) {
    return scan1d_rss(Kind::I32, x, y, n, ws, ws_bytes, stream);
}
int scan_inclusive_rss_f32(const float* x, float* y, int64_t n, void* ws, size_t ws_bytes,
                           void* stream) {
    return scan1d_rss(Kind::F32, x, y, n, ws, ws_bytes, stream);
}

int scan_rows_i32(const int32_t* x, int32_t* y, int64_t rows, int64_t len, int exclusive, void* ws,
                  size_t ws_bytes, void* stream) {
    return scan_rows(Kind::I32, x, y, rows, len, exclusive, ws, ws_bytes, stream);
}
int scan_rows_f32(const float* x, float* y, int64_t rows, int64_t len, int exclusive, void* ws,
                  size_t ws_bytes, void* stream) {
    return scan_rows(Kind::F32, x, y, rows, len, exclusive, ws, ws_bytes, stream);
}

int topp_cutoff_f32(const float* probs, int32_t* cutoff, int64_t rows, int64_t len, float p,
                    void* ws, size_t ws_bytes, void* stream) {
    const int r = check_rows(rows, len);
    if (r != LIBSCAN_OK) return r;
    if (len > INT32_MAX) return LIBSCAN_ERANGE;
    if (p != p) return LIBSCAN_EINVAL;  // NaN
    if (rows > 0 && !cutoff) return LIBSCAN_EINVAL;
    const size_t bytes = (size_t)rows * (size_t)len * 4;
    if (bytes > 0 && !probs) return LIBSCAN_EINVAL;
    if (overlaps(probs, bytes, cutoff, (size_t)rows * 4)) return LIBSCAN_EINVAL;
    if (rows == 0) return LIBSCAN_OK;
    const int w = check_ws(ws, ws_bytes, ls::scan_rows_ws_bytes(rows, len));
    if (w != LIBSCAN_OK) return w;
    return hip_status(ls::launch_topp_cutoff(probs, cutoff, rows, len, p, ws, ws_bytes,
                                             (hipStream_t)stream));
}

int compact_by_mask_f32(const float* x, const uint8_t* mask, float* out, int32_t* idx_out,
                        int32_t* count_dev, int64_t n, void* ws, size_t ws_bytes, void* stream) {
    if (n < 0 || !count_dev) return LIBSCAN_EINVAL;
    if (n > INT32_MAX) return LIBSCAN_ERANGE;
    if (n > 0 && (!x || !mask || !out)) return LIBSCAN_EINVAL;
    const size_t b4 = (size_t)n * 4, b1 = (size_t)n;
    if (overlaps(out, b4, x, b4) || overlaps(out, b4, mask, b1) || overlaps(out, b4, count_dev, 4) ||
        overlaps(idx_out, b4, x, b4) || overlaps(idx_out, b4, mask, b1) ||
        overlaps(idx_out, b4, out, b4) || overlaps(idx_out, b4, count_dev, 4) ||
        overlaps(count_dev, 4, x, b4) || overlaps(count_dev, 4, mask, b1))
        return LIBSCAN_EINVAL;
    if (n > 0) {
        const int w = check_ws(ws, ws_bytes, ls::compact_ws_bytes(n));
        if (w != LIBSCAN_OK) return w;
    }
    return hip_status(ls::launch_compact(x, mask, out, idx_out, count_dev, n, ws, ws_bytes,
                                         (hipStream_t)stream));
}

int split_by_flags_u32(const uint32_t* keys, const int32_t* idx_in, const uint8_t* flags,
                       uint32_t* keys_out, int32_t* idx_out, int32_t* n_true_dev, int64_t n,
                       void* ws, size_t ws_bytes, void* stream) {
    if (n < 0) return LIBSCAN_EINVAL;
    if (n > INT32_MAX) return LIBSCAN_ERANGE;
    if (n > 0 && (!keys || !flags || !keys_out)) return LIBSCAN_EINVAL;
    const size_t b4 = (size_t)n * 4, b1 = (size_t)n;
    const void* ins[3] = {keys, idx_in, flags};
    const size_t inb[3] = {b4, idx_in ? b4 : 0, b1};
    void* outs[3] = {keys_out, idx_out, n_true_dev};
    const size_t outb[3] = {b4, idx_out ? b4 : 0, n_true_dev ? 4u : 0u};
    for (int o = 0; o < 3; ++o) {
        for (int i = 0; i < 3; ++i)
            if (overlaps(outs[o], outb[o], ins[i], inb[i])) return LIBSCAN_EINVAL;
        for (int p = o + 1; p < 3; ++p)
            if (overlaps(outs[o], outb[o], outs[p], outb[p])) return LIBSCAN_EINVAL;
    }
    if (n > 0) {
        const int w = check_ws(ws, ws_bytes, ls::compact_ws_bytes(n));
        if (w != LIBSCAN_OK) return w;
    } else if (!n_true_dev) {
        return LIBSCAN_OK;
    }
    return hip_status(ls::launch_split(keys, idx_in, flags, 0, keys_out, idx_out, n_true_dev, n, ws,
                                       ws_bytes, (hipStream_t)stream));
}

int radix_sort_u32(const uint32_t* keys, uint32_t* keys_out, int32_t* perm_out, uint32_t* keys_tmp,
                   int32_t* perm_tmp, int64_t n, int bits_per_pass, void* ws, size_t ws_bytes,
                   void* stream) {
    if (n < 0 || (bits_per_pass != 1 && bits_per_pass != 4 && bits_per_pass != 8))
        return LIBSCAN_EINVAL;
    if (n > ls::kMaxRadixKeys) return LIBSCAN_ERANGE;
    if (n == 0) return LIBSCAN_OK;
    if (!keys || !keys_out || !keys_tmp || (perm_out && !perm_tmp)) return LIBSCAN_EINVAL;
    const size_t b = (size_t)n * 4;
    const void* bufs[5] = {keys, keys_out, perm_out, keys_tmp, perm_out ? perm_tmp : nullptr};
    for (int i = 0; i < 5; ++i)
        for (int j = i + 1; j < 5; ++j)
            if (overlaps(bufs[i], bufs[i] ? b : 0, bufs[j], bufs[j] ? b : 0)) return LIBSCAN_EINVAL;
    const int w = check_ws(ws, ws_bytes, ls::radix_ws_bytes(n, bits_per_pass));
    if (w != LIBSCAN_OK) return w;
    return hip_status(ls::launch_radix_sort(keys, keys_out, perm_out, keys_tmp, perm_tmp, n,
                                            bits_per_pass, ws, ws_bytes, (hipStream_t)stream));
}

int radix_sort_i32(const int32_t* keys, int32_t* keys_out, int32_t* perm_out, int32_t* keys_tmp,
                   int32_t* perm_tmp, int64_t n, int descending, void* ws, size_t ws_bytes,
                   void* stream) {
    return radix_sort_typed(ls::KeyType::I32, 4, keys, keys_out, perm_out, keys_tmp, perm_tmp, n,
                            descending, ws, ws_bytes, stream);
}

int radix_sort_f32(const float* keys, float* keys_out, int32_t* perm_out, float* keys_tmp,
                   int32_t* perm_tmp, int64_t n, int descending, void* ws, size_t ws_bytes,
                   void* stream) {
    return radix_sort_typed(ls::KeyType::F32, 4, keys, keys_out, perm_out, keys_tmp, perm_tmp, n,
                            descending, ws, ws_bytes, stream);
}

int radix_sort_f16(const uint16_t* keys, uint16_t* keys_out, int32_t* perm_out, uint16_t* keys_tmp,
                   int32_t* perm_tmp, int64_t n, int descending, void* ws, size_t ws_bytes,
                   void* stream) {
    return radix_sort_typed(ls::KeyType::F16, 2, keys, keys_out, perm_out, keys_tmp, perm_tmp, n,
                            descending, ws, ws_bytes, stream);
}

int radix_sort_rows_f32(const float* keys, float* keys_out, int32_t* perm_out, float* keys_tmp,
                        int32_t* perm_tmp, int64_t rows, int64_t len, int descending, void* ws,
                        size_t ws_bytes, void* stream) {
    if (rows < 0 || len < 0) return LIBSCAN_EINVAL;
    if (!ls::radix_rows_fit(rows, len)) return LIBSCAN_ERANGE;
    if (rows == 0 || len == 0) return LIBSCAN_OK;
    if (!keys || !keys_out || !keys_tmp || (perm_out && !perm_tmp)) return LIBSCAN_EINVAL;
    const size_t b = (size_t)rows * (size_t)len * 4;
    const void* bufs[5] = {keys, keys_out, perm_out, keys_tmp, perm_out ? perm_tmp : nullptr};
    for (int i = 0; i < 5; ++i)
        for (int j = i + 1; j < 5; ++j)
            if (overlaps(bufs[i], bufs[i] ? b : 0, bufs[j], bufs[j] ? b : 0)) return LIBSCAN_EINVAL;
    const int w = check_ws(ws, ws_bytes, ls::radix_rows_ws_bytes(rows, len));
    if (w != LIBSCAN_OK) return w;
    return hip_status(ls::launch_radix_sort_typed(ls::KeyType::F32, descending != 0, keys,
                                                  keys_out, nullptr, perm_out, keys_tmp, perm_tmp,
                                                  rows, len, ws, ws_bytes, (hipStream_t)stream));
}

int weighted_sample_f32(const float* w, const float* theta_dev, int32_t* out, int64_t rows,
                        int64_t len, void* ws, size_t ws_bytes, void* stream) {
    const int c = check_sample(w, theta_dev, out, nullptr, rows, len);
    if (c != LIBSCAN_OK || rows == 0) return c;
    const int k = check_ws(ws, ws_bytes, ls::weighted_ws_bytes(rows, len));
    if (k != LIBSCAN_OK) return k;
    return hip_status(ls::launch_weighted_sample(w, theta_dev, out, rows, len, ws,
                                                 (hipStream_t)stream));
}

int topp_sample_f32(const float* probs, const float* theta_dev, float p, int32_t* token_out,
                    int32_t* cutoff_out, int64_t rows, int64_t len, void* scratch,
                    size_t scratch_bytes, void* ws, size_t ws_bytes, void* stream) {
    if (p != p) return LIBSCAN_EINVAL;  // NaN
    const int c = check_sample(probs, theta_dev, token_out, cutoff_out, rows, len);
    if (c != LIBSCAN_OK) return c;
    if (!ls::radix_rows_fit(rows, len)) return LIBSCAN_ERANGE;
    if (rows == 0) return LIBSCAN_OK;
    const size_t need = ls::topp_sample_scratch_bytes(rows, len);
    if (len > 0) {
        if (scratch_bytes < need) return LIBSCAN_ENOSPACE;
        if (!scratch || ((uintptr_t)scratch % 16) != 0) return LIBSCAN_EINVAL;
        const size_t xb = (size_t)rows * (size_t)len * 4, rb = (size_t)rows * 4;
        if (overlaps(scratch, need, probs, xb) || overlaps(scratch, need, theta_dev, rb) ||
            overlaps(scratch, need, token_out, rb) ||
            overlaps(scratch, need, cutoff_out, cutoff_out ? rb : 0) ||
            overlaps(scratch, need, ws, ws_bytes))
            return LIBSCAN_EINVAL;
    }
    const int k = check_ws(ws, ws_bytes, ls::topp_sample_ws_bytes(rows, len));
    if (k != LIBSCAN_OK) return k;
    return hip_status(ls::launch_topp_sample(probs, theta_dev, p, token_out, cutoff_out, rows, len,
                                             scratch, ws, (hipStream_t)stream));
}

int topk_rows_f32(const float* x, float* values_out, int32_t* idx_out, int64_t rows, int64_t len,
                  int64_t k, int largest, void* scratch, size_t scratch_bytes, void* ws,
                  size_t ws_bytes, void* stream) {
    const int r = check_topk(rows, len, k);
    if (r != LIBSCAN_OK) return r;
    if (rows == 0 || k == 0) return LIBSCAN_OK;
    if (!x || !values_out || !idx_out) return LIBSCAN_EINVAL;
    const size_t xb = (size_t)rows * (size_t)len * 4, ob = (size_t)rows * (size_t)k * 4;
    const size_t need = ls::topk_scratch_bytes(rows, len, k);
    if (scratch_bytes < need) return LIBSCAN_ENOSPACE;
    if (!scratch || ((uintptr_t)scratch % 16) != 0) return LIBSCAN_EINVAL;
    if (overlaps(values_out, ob, x, xb) || overlaps(idx_out, ob, x, xb) ||
        overlaps(values_out, ob, idx_out, ob) || overlaps(scratch, need, x, xb) ||
        overlaps(scratch, need, values_out, ob) || overlaps(scratch, need, idx_out, ob) ||
        overlaps(scratch, need, ws, ws_bytes))
        return LIBSCAN_EINVAL;
    const int w = check_ws(ws, ws_bytes, ls::topk_ws_bytes(rows, len, k));
    if (w != LIBSCAN_OK) return w;
    return hip_status(ls::launch_topk(x, values_out, idx_out, rows, len, k, largest != 0, scratch,
                                      ws, (hipStream_t)stream));
}

int libscan_scratch_bytes(int op, int64_t rows, int64_t len, int64_t k, size_t* bytes) {
    if (!bytes || rows < 0 || len < 0 || k < 0) return LIBSCAN_EINVAL;
    switch (op) {
        case LIBSCAN_OP_TOPP_SAMPLE: {
            const int r = check_rows(rows, len);
            if (r != LIBSCAN_OK) return r;
            if (!ls::radix_rows_fit(rows, len)) return LIBSCAN_ERANGE;
            *bytes = ls::topp_sample_scratch_bytes(rows, len);
            return LIBSCAN_OK;
        }
        case LIBSCAN_OP_TOPK: {
            const int r = check_topk(rows, len, k);
            if (r != LIBSCAN_OK) return r;
            *bytes = ls::topk_scratch_bytes(rows, len, k);
            return LIBSCAN_OK;
        }
        default:
            return LIBSCAN_EINVAL;
    }
}

}  // extern "C"
