// noalloc.hip -- the inclusive int32 scan without a caller workspace, for
// callers that cannot allocate device memory (code under HIP graph capture,
// tight serving loops, harnesses that forbid hipMalloc).
//
// The look-back kernels need a workspace (ticket header + one status word per
// tile).  Here it is a file-scope device array of fixed size, one copy per
// GPU, kept until the process ends.  Host code never uses the array's name as
// an address: at the first call on a device (with that device current) the
// device address of that GPU's copy is looked up once with
// hipGetSymbolAddress and kept per device, and that pointer is what the
// kernels receive.  The same first call zero-fills the array with a fill
// kernel on the caller's stream (a zero-filled workspace is ready, and the
// epoch-tagged protocol keeps it ready for every later call, so nothing is
// cleared again).  Nothing here calls hipMalloc, hipFree or any allocating
// routine.
#include <mutex>

#include "../../include/libscan.h"
#include "launch.hpp"

namespace {

// Workspace of a 1-D scan of up to LIBSCAN_NOALLOC_MAX_N elements: the
// 256-byte header plus one 8-byte status word per smallest (4096-element)
// tile, i.e. 4 MiB + 256 bytes.
constexpr int64_t kMaxN = LIBSCAN_NOALLOC_MAX_N;
constexpr size_t kScratchBytes = ls::kWsHeader + (size_t)((kMaxN + 4095) / 4096) * 8;
static_assert(kScratchBytes % 256 == 0, "scratch is a whole number of 256-byte blocks");

}  // namespace

// One copy per GPU.  In host code this name is only the host-side stand-in of
// the array, never a device address: kernels get g_ptr[dev] below.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_mutex;
void* g_ptr[kMaxDevices];  // device address of `scratch` on each GPU, once looked up

// The current device's copy of `scratch`, set up on first use (looked up and
// zero-filled on `stream`).  nullptr on a HIP error.
void* device_scratch(hipStream_t stream) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_mutex);
    if (g_ptr[dev]) return g_ptr[dev];
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
    if (ls::launch_workspace_init(p, kScratchBytes, stream) != hipSuccess) return nullptr;
    g_ptr[dev] = p;
    return p;
}

}  // namespace

extern "C" int scan_inclusive_i32_noalloc(const int32_t* x, int32_t* y, int64_t n, void* stream) {
    if (n < 0) return LIBSCAN_EINVAL;
    if (n > kMaxN) return LIBSCAN_ERANGE;
    if (n > 0 && (!x || !y)) return LIBSCAN_EINVAL;
    const uintptr_t x0 = (uintptr_t)x, y0 = (uintptr_t)y, b = (uintptr_t)n * 4;
    if (n > 0 && x0 != y0 && x0 < y0 + b && y0 < x0 + b) return LIBSCAN_EINVAL;  // partial overlap
    if (n == 0) return LIBSCAN_OK;
    hipStream_t s = (hipStream_t)stream;
    void* ws = device_scratch(s);
    if (!ws) return LIBSCAN_EHIP;
    const hipError_t e = ls::launch_scan1d(ls::Kind::I32, false, x, y, n, nullptr, nullptr, ws,
                                           kScratchBytes, s);
    return e == hipSuccess ? LIBSCAN_OK : LIBSCAN_EHIP;
}
