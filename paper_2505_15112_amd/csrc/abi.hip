// abi.hip -- the extern "C" entry points of libscan (declared in libscan.h).
//
// Each entry point checks its arguments on the host, before any HIP call, and
// then enqueues the kernels through the launchers of launch.hpp.
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

int libscan_workspace_bytes(int op, int64_t n, int64_t rows, int64_t len, int bits, size_t* bytes) {
    (void)bits;
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

}  // extern "C"
