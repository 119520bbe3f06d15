// launch.hpp -- internal host-side launchers behind the C ABI.
//
// Every launcher enqueues kernels on `stream` and returns the launch status;
// the C ABI validates arguments before calling any of these.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ls {

// Element kinds of the 1-D scans: input type -> accumulation/output type.
enum class Kind { I32, F32, F16F32, U8I32 };

constexpr size_t kWsHeader = 256;  // counters at the front of every workspace
constexpr int64_t kMaxScanElems = int64_t(1) << 35;

// Zero-fill a workspace (its first use; see WsHeader in device.hpp).
hipError_t launch_workspace_init(void* ws, size_t ws_bytes, hipStream_t stream);

// 1-D decoupled look-back scan.
size_t scan1d_ws_bytes(int64_t n);
hipError_t launch_scan1d(Kind kind, bool exclusive, const void* x, void* y, int64_t n,
                         const void* carry_in, void* total_out, void* ws, size_t ws_bytes,
                         hipStream_t stream);

// 1-D reduce-then-scan (three kernels).
size_t scan1d_rss_ws_bytes(int64_t n);
hipError_t launch_scan1d_rss(Kind kind, const void* x, void* y, int64_t n, void* ws,
                             hipStream_t stream);

}  // namespace ls
