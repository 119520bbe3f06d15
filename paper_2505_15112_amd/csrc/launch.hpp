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
// Copy the workspace's error word into *out (device int32), clearing it if reset.
hipError_t launch_workspace_error(void* ws, int32_t* out, bool reset, hipStream_t stream);

// 1-D decoupled look-back scan: launch_scan1d picks the kernel (the
// matrix-core one for inclusive fp16 scans of at least one whole tile),
// launch_scan1d_tiles always the wavefront tiles.
size_t scan1d_ws_bytes(int64_t n);
hipError_t launch_scan1d(Kind kind, bool exclusive, const void* x, void* y, int64_t n,
                         const void* carry_in, void* total_out, void* ws, size_t ws_bytes,
                         hipStream_t stream);
hipError_t launch_scan1d_tiles(Kind kind, bool exclusive, const void* x, void* y, int64_t n,
                               const void* carry_in, void* total_out, void* ws, size_t ws_bytes,
                               hipStream_t stream);

// 1-D inclusive scan of fp16 with the tile-local row scans on the matrix
// cores (ScanU) on whole tiles of kMfmaTileElems, the tail on the wavefront
// tiles; same workspace as launch_scan1d.  x 16-byte aligned.
constexpr int64_t kMfmaTileElems = 32768;
hipError_t launch_scan1d_mfma_f16(const uint16_t* x, float* y, int64_t n, void* ws,
                                  size_t ws_bytes, hipStream_t stream);
// The exclusive byte scan the same way (v_mfma_i32_32x32x32_i8); total_out
// (nullable) gets the sum of all bytes.  x 16-byte aligned.
hipError_t launch_scan1d_mfma_u8(const uint8_t* x, uint32_t* y, int64_t n, uint32_t* total_out,
                                 void* ws, size_t ws_bytes, hipStream_t stream);

// 1-D reduce-then-scan (three kernels).
size_t scan1d_rss_ws_bytes(int64_t n);
hipError_t launch_scan1d_rss(Kind kind, const void* x, void* y, int64_t n, void* ws,
                             hipStream_t stream);

// Batched row scans (rows x len, row-major) and the top-p cutoff on them.
size_t scan_rows_ws_bytes(int64_t rows, int64_t len);
hipError_t launch_scan_rows(Kind kind, bool exclusive, const void* x, void* y, int64_t rows,
                            int64_t len, void* ws, size_t ws_bytes, hipStream_t stream);
size_t topp_ws_bytes(int64_t rows, int64_t len);
size_t weighted_ws_bytes(int64_t rows, int64_t len);
bool radix_rows_fit(int64_t rows, int64_t len);
size_t topp_sample_ws_bytes(int64_t rows, int64_t len);
size_t topp_sample_scratch_bytes(int64_t rows, int64_t len);
size_t topk_ws_bytes(int64_t rows, int64_t len, int64_t k);
size_t topk_scratch_bytes(int64_t rows, int64_t len, int64_t k);
hipError_t launch_topk(const float* x, float* values, int32_t* indices, int64_t rows, int64_t len,
                       int64_t k, bool largest, void* scratch, void* ws, hipStream_t stream);
hipError_t launch_topp_sample(const float* probs, const float* theta, float p, int32_t* token,
                              int32_t* cutoff, int64_t rows, int64_t len, void* scratch, void* ws,
                              hipStream_t stream);
hipError_t launch_weighted_sample(const float* w, const float* theta, int32_t* out, int64_t rows,
                                  int64_t len, void* ws, hipStream_t stream);
hipError_t launch_topp_draw_sorted(const float* sorted, const int32_t* idx, const float* theta,
                                   float p, int32_t* token, int32_t* cutoff, int64_t rows,
                                   int64_t len, void* ws, hipStream_t stream);
hipError_t launch_topp_cutoff(const float* probs, int32_t* cutoff, int64_t rows, int64_t len,
                              float p, void* ws, size_t ws_bytes, hipStream_t stream);
constexpr int64_t kMaxGridTiles = int64_t(1) << 24;
// Radix sorts: keys per call (rows x len in total), indices being int32.
constexpr int64_t kMaxRadixKeys = INT32_MAX;

// Compress and split (Section 5).  flags == nullptr in launch_split means
// "flag = key bit `bit` is 0" (the LSB radix-sort pass).
size_t compact_ws_bytes(int64_t n);
hipError_t launch_compact(const float* x, const uint8_t* mask, float* out, int32_t* idx,
                          int32_t* count, int64_t n, void* ws, size_t ws_bytes,
                          hipStream_t stream);
hipError_t launch_split(const uint32_t* keys, const int32_t* idx_in, const uint8_t* flags, int bit,
                        uint32_t* keys_out, int32_t* idx_out, int32_t* n_true_out, int64_t n,
                        void* ws, size_t ws_bytes, hipStream_t stream);

// Key types of the typed radix sorts (8-bit digits; encoded on the first pass,
// decoded on the last).
enum class KeyType { U32, I32, F32, F16 };
// rows = 1: a 1-D sort of len keys; else every row of a rows x len matrix on
// its own (perm_out: indices within the row).  perm_in (nullable, needs
// perm_out): the index carried by each key instead of its position.
hipError_t launch_radix_sort_typed(KeyType type, bool descending, const void* keys,
                                   void* keys_out, const int32_t* perm_in, int32_t* perm_out,
                                   void* keys_tmp,
                                   int32_t* perm_tmp, int64_t rows, int64_t len, void* ws,
                                   size_t ws_bytes, hipStream_t stream);
size_t radix_rows_ws_bytes(int64_t rows, int64_t len);

// LSD radix sort (1, 4 or 8 bits per pass), caller-provided ping-pong buffers.
size_t radix_ws_bytes(int64_t n, int bits);
hipError_t launch_radix_sort(const uint32_t* keys, uint32_t* keys_out, int32_t* perm_out,
                             uint32_t* keys_tmp, int32_t* perm_tmp, int64_t n, int bits, void* ws,
                             size_t ws_bytes, hipStream_t stream);

}  // namespace ls
