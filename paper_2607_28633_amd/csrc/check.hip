// check.hip - checked path of libtopkv.so: device-side validation of block
// tables and lengths, and of fixed-state slot indices (declared in
// include/topkv.h), and checked mode (TOPKV_CHECKED=1), which runs that
// validation inside the movement calls.  The movement kernels never depend on
// it; they bounds-check what they read and skip bad entries silently, and
// these calls report them.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdlib>
#include <mutex>
#include <vector>

#include "internal.h"
#include "topkv.h"

namespace {

// result[0] status, [1] entries outside [0, num_pages), [2] pages named more
// than once, [3] lengths outside [0, bt_stride * page_size].
__global__ __launch_bounds__(256) void kv_check_clear_kernel(uint32_t* __restrict__ bitmap, int64_t words,
                                                             int32_t* __restrict__ result) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t w = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; w < words; w += stride) bitmap[w] = 0u;
  if (blockIdx.x == 0 && threadIdx.x < 4) result[threadIdx.x] = 0;
}

// One thread per (request, table entry) slot.  With a window (> 0) only the
// pages holding the last `window` tokens are read by a move, so only their
// entries are checked.
__global__ __launch_bounds__(256) void kv_check_tables_kernel(const int32_t* __restrict__ tables,
                                                              const int32_t* __restrict__ seq_lens,
                                                              int32_t num_reqs, int32_t bt_stride,
                                                              int32_t page_size, int64_t num_pages,
                                                              int32_t window, int32_t check_duplicates,
                                                              uint32_t* __restrict__ bitmap,
                                                              int32_t* __restrict__ result) {
  const int64_t slot = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (slot >= (int64_t)num_reqs * bt_stride) return;
  const int32_t r = (int32_t)(slot / bt_stride);
  const int32_t i = (int32_t)(slot - (int64_t)r * bt_stride);
  int64_t n = seq_lens[r];
  const int64_t max_tok = (int64_t)bt_stride * page_size;
  if (n < 0 || n > max_tok) {
    if (i == 0) atomicAdd(&result[3], 1);
    n = n < 0 ? 0 : max_tok;
  }
  if ((int64_t)i * page_size >= n) return;     // past the request's last page: never read
  const int64_t start = (window > 0 && n > window) ? n - window : 0;
  if ((int64_t)(i + 1) * page_size <= start) return;   // before the window: never read
  const int32_t e = tables[slot];
  if (e < 0 || (int64_t)e >= num_pages) {
    atomicAdd(&result[1], 1);
    return;
  }
  if (check_duplicates) {
    const uint32_t bit = 1u << (e & 31);
    const uint32_t old = atomicOr(&bitmap[e >> 5], bit);
    if (old & bit) atomicAdd(&result[2], 1);
  }
}

// One thread per request of a fixed-state layer batch: its slot must lie in
// [0, num_slots) and, with check_duplicates, no slot may be named twice.
__global__ __launch_bounds__(256) void kv_check_slots_kernel(const int32_t* __restrict__ slots, int32_t num_reqs,
                                                             int64_t num_slots, int32_t check_duplicates,
                                                             uint32_t* __restrict__ bitmap,
                                                             int32_t* __restrict__ result) {
  const int32_t r = (int32_t)(blockIdx.x * blockDim.x + threadIdx.x);
  if (r >= num_reqs) return;
  const int32_t e = slots[r];
  if (e < 0 || (int64_t)e >= num_slots) {
    atomicAdd(&result[1], 1);
    return;
  }
  if (check_duplicates) {
    const uint32_t bit = 1u << (e & 31);
    const uint32_t old = atomicOr(&bitmap[e >> 5], bit);
    if (old & bit) atomicAdd(&result[2], 1);
  }
}

__global__ void kv_check_finish_kernel(int32_t* __restrict__ result) {
  if (threadIdx.x == 0)
    result[0] = (result[1] | result[2] | result[3]) ? (int32_t)TOPKV_ERR_BOUNDS : (int32_t)TOPKV_OK;
}

// Clear, per-slot check and verdict on `stream` (the arguments validated by
// the caller).
topkv_status_t launch_table_check(const topkv_pool_t* pool, int32_t num_reqs, const int32_t* block_tables,
                                  int32_t bt_stride, const int32_t* seq_lens, int32_t window, bool dup,
                                  uint32_t* bitmap, int32_t* result, hipStream_t stream) {
  const int64_t clear_words = dup ? (pool->num_pages + 31) / 32 : 0;
  const unsigned clear_grid = (unsigned)(clear_words / 256 + 1 < 1024 ? clear_words / 256 + 1 : 1024);
  hipLaunchKernelGGL(kv_check_clear_kernel, dim3(clear_grid), dim3(256), 0, stream, dup ? bitmap : nullptr,
                     clear_words, result);
  if (hipGetLastError() != hipSuccess) return TOPKV_ERR_LAUNCH;
  const int64_t slots = (int64_t)num_reqs * bt_stride;
  if (slots > 0) {
    if (slots / 256 + 1 > INT32_MAX) return TOPKV_ERR_UNSUPPORTED;
    hipLaunchKernelGGL(kv_check_tables_kernel, dim3((unsigned)((slots + 255) / 256)), dim3(256), 0, stream,
                       block_tables, seq_lens, num_reqs, bt_stride, pool->page_size, pool->num_pages, window,
                       (int32_t)dup, bitmap, result);
    if (hipGetLastError() != hipSuccess) return TOPKV_ERR_LAUNCH;
  }
  hipLaunchKernelGGL(kv_check_finish_kernel, dim3(1), dim3(64), 0, stream, result);
  return hipGetLastError() == hipSuccess ? TOPKV_OK : TOPKV_ERR_LAUNCH;
}

// Checked mode's device buffer, one per device: result int32[4] at 0, a
// host-side length staged at 16, the page or slot bitmap from 64.  Allocated
// on first use and grown on demand; kept until the process ends.  The lock
// is held from the check's first launch to the stream synchronisation.
constexpr int kMaxDevices = 64;
constexpr int64_t kLenOffset = 16;
constexpr int64_t kBitmapOffset = 64;

struct CheckBuffer {
  std::mutex mu;
  char* ptr = nullptr;
  int64_t bytes = 0;
};
CheckBuffer g_check[kMaxDevices];

topkv_status_t grow(CheckBuffer& b, int64_t bytes) {
  if (b.bytes >= bytes) return TOPKV_OK;
  if (b.ptr && hipFree(b.ptr) != hipSuccess) return TOPKV_ERR_DEVICE;
  b.ptr = nullptr;
  b.bytes = 0;
  const int64_t want = bytes < 4096 ? 4096 : bytes;
  void* p = nullptr;
  if (hipMalloc(&p, (size_t)want) != hipSuccess) return TOPKV_ERR_DEVICE;
  b.ptr = static_cast<char*>(p);
  b.bytes = want;
  return TOPKV_OK;
}

// Checked mode synchronises, so it refuses streams under capture.
topkv_status_t check_stream(hipStream_t stream, int* dev) {
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(stream, &cs) != hipSuccess) return TOPKV_ERR_DEVICE;
  if (cs != hipStreamCaptureStatusNone) return TOPKV_ERR_UNSUPPORTED;
  if (hipGetDevice(dev) != hipSuccess || *dev < 0) return TOPKV_ERR_DEVICE;
  return *dev < kMaxDevices ? TOPKV_OK : TOPKV_ERR_UNSUPPORTED;
}

}  // namespace

namespace topkv_internal {

bool checked_mode() {
  const char* e = std::getenv("TOPKV_CHECKED");
  return e && e[0] == '1' && e[1] == '\0';
}

topkv_status_t checked_tables(const topkv_pool_t* pool, int32_t num_reqs, const int32_t* block_tables,
                              int32_t bt_stride, const int32_t* seq_lens, int32_t seq_len, int32_t window,
                              bool duplicates, int64_t per_token, int64_t fixed_bytes, int64_t packed_cap,
                              hipStream_t stream) {
  int dev = 0;
  topkv_status_t st = check_stream(stream, &dev);
  if (st != TOPKV_OK) return st;
  if (num_reqs <= 0) return TOPKV_OK;
  if ((int64_t)bt_stride * pool->page_size > INT32_MAX) return TOPKV_ERR_UNSUPPORTED;
  CheckBuffer& b = g_check[dev];
  std::lock_guard<std::mutex> lock(b.mu);
  const int64_t words = duplicates ? (pool->num_pages + 31) / 32 : 0;
  st = grow(b, kBitmapOffset + 4 * words);
  if (st != TOPKV_OK) return st;
  int32_t* result = reinterpret_cast<int32_t*>(b.ptr);
  const int32_t* lens = seq_lens;
  if (!seq_lens) {                                    // one request with a host-side length
    int32_t* staged = reinterpret_cast<int32_t*>(b.ptr + kLenOffset);
    if (hipMemcpyAsync(staged, &seq_len, sizeof(int32_t), hipMemcpyHostToDevice, stream) != hipSuccess)
      return TOPKV_ERR_DEVICE;
    lens = staged;
  }
  int32_t res[4] = {0, 0, 0, 0};
  std::vector<int32_t> host(seq_lens ? (size_t)num_reqs : 1, seq_len);
  st = launch_table_check(pool, num_reqs, block_tables, bt_stride, lens, window, duplicates,
                          reinterpret_cast<uint32_t*>(b.ptr + kBitmapOffset), result, stream);
  if (st == TOPKV_OK && hipMemcpyAsync(res, result, sizeof(res), hipMemcpyDeviceToHost, stream) != hipSuccess)
    st = TOPKV_ERR_DEVICE;
  if (st == TOPKV_OK && seq_lens &&
      hipMemcpyAsync(host.data(), seq_lens, sizeof(int32_t) * (size_t)num_reqs, hipMemcpyDeviceToHost, stream) !=
          hipSuccess)
    st = TOPKV_ERR_DEVICE;
  // Whatever was queued (the staged length's copy included) completes before
  // this frame and the buffer's lock go away, also on the failure paths.
  if (hipStreamSynchronize(stream) != hipSuccess && st == TOPKV_OK) st = TOPKV_ERR_DEVICE;
  if (st != TOPKV_OK) return st;
  if (res[0] != TOPKV_OK) return TOPKV_ERR_BOUNDS;
  // The packed buffer must hold every kept token (a batched request that
  // would cross its end is otherwise left unmoved); lengths are in range here.
  int64_t kept = 0;
  for (const int32_t n : host) kept += (window > 0 && n > window) ? window : n;
  int64_t need;
  if (kept > 0 && (__builtin_mul_overflow(kept, per_token, &need) ||
                   __builtin_add_overflow(need, fixed_bytes, &need) || need > packed_cap))
    return TOPKV_ERR_BOUNDS;
  return TOPKV_OK;
}

topkv_status_t checked_slots(const topkv_state_pool_t* pool, int32_t num_reqs, const int32_t* slots,
                             bool duplicates, hipStream_t stream) {
  int dev = 0;
  topkv_status_t st = check_stream(stream, &dev);
  if (st != TOPKV_OK) return st;
  if (num_reqs <= 0) return TOPKV_OK;
  CheckBuffer& b = g_check[dev];
  std::lock_guard<std::mutex> lock(b.mu);
  const int64_t words = duplicates ? (pool->num_slots + 31) / 32 : 0;
  st = grow(b, kBitmapOffset + 4 * words);
  if (st != TOPKV_OK) return st;
  int32_t* result = reinterpret_cast<int32_t*>(b.ptr);
  int32_t res[4] = {0, 0, 0, 0};
  st = topkv_check_state_slots(pool, num_reqs, slots, duplicates ? 1 : 0, b.ptr + kBitmapOffset, 4 * words, result,
                               stream);
  if (st == TOPKV_OK && hipMemcpyAsync(res, result, sizeof(res), hipMemcpyDeviceToHost, stream) != hipSuccess)
    st = TOPKV_ERR_DEVICE;
  if (hipStreamSynchronize(stream) != hipSuccess && st == TOPKV_OK) st = TOPKV_ERR_DEVICE;
  if (st != TOPKV_OK) return st;
  return res[0] == TOPKV_OK ? TOPKV_OK : TOPKV_ERR_BOUNDS;
}

}  // namespace topkv_internal

extern "C" {

int64_t topkv_check_workspace_bytes(const topkv_pool_t* pool) {
  if (!pool || pool->num_pages <= 0) return -1;
  return ((pool->num_pages + 31) / 32) * (int64_t)sizeof(uint32_t);
}

topkv_status_t topkv_check_tables(const topkv_pool_t* pool, int32_t num_reqs, const int32_t* block_tables,
                                  int32_t bt_stride, const int32_t* seq_lens, int32_t check_duplicates,
                                  void* workspace, int64_t workspace_bytes, int32_t* result,
                                  hipStream_t stream) {
  if (!pool || pool->num_pages <= 0 || pool->page_size <= 0 || num_reqs < 0 || !result) return TOPKV_ERR_INVALID_ARG;
  if (num_reqs > 0 && (!block_tables || !seq_lens || bt_stride <= 0)) return TOPKV_ERR_INVALID_ARG;
  if ((int64_t)bt_stride * pool->page_size > INT32_MAX) return TOPKV_ERR_UNSUPPORTED;
  const int64_t words = (pool->num_pages + 31) / 32;
  const bool dup = check_duplicates != 0;
  if (dup && (!workspace || workspace_bytes < words * (int64_t)sizeof(uint32_t))) return TOPKV_ERR_INVALID_ARG;
  return launch_table_check(pool, num_reqs, block_tables, bt_stride, seq_lens, 0, dup,
                            static_cast<uint32_t*>(workspace), result, stream);
}

int64_t topkv_check_state_workspace_bytes(const topkv_state_pool_t* pool) {
  if (!pool || pool->num_slots <= 0) return -1;
  return ((pool->num_slots + 31) / 32) * (int64_t)sizeof(uint32_t);
}

topkv_status_t topkv_check_state_slots(const topkv_state_pool_t* pool, int32_t num_reqs, const int32_t* slots,
                                       int32_t check_duplicates, void* workspace, int64_t workspace_bytes,
                                       int32_t* result, hipStream_t stream) {
  if (!pool || pool->num_slots <= 0 || num_reqs < 0 || !result || (num_reqs > 0 && !slots))
    return TOPKV_ERR_INVALID_ARG;
  const int64_t words = (pool->num_slots + 31) / 32;
  const bool dup = check_duplicates != 0;
  if (dup && (!workspace || workspace_bytes < words * (int64_t)sizeof(uint32_t))) return TOPKV_ERR_INVALID_ARG;
  uint32_t* bitmap = dup ? static_cast<uint32_t*>(workspace) : nullptr;
  const int64_t clear_words = dup ? words : 0;
  const unsigned clear_grid = (unsigned)(clear_words / 256 + 1 < 1024 ? clear_words / 256 + 1 : 1024);
  hipLaunchKernelGGL(kv_check_clear_kernel, dim3(clear_grid), dim3(256), 0, stream, bitmap, clear_words,
                     result);
  if (hipGetLastError() != hipSuccess) return TOPKV_ERR_LAUNCH;
  if (num_reqs > 0) {
    hipLaunchKernelGGL(kv_check_slots_kernel, dim3((unsigned)(((int64_t)num_reqs + 255) / 256)), dim3(256), 0, stream,
                       slots, num_reqs, pool->num_slots, (int32_t)dup, bitmap, result);
    if (hipGetLastError() != hipSuccess) return TOPKV_ERR_LAUNCH;
  }
  hipLaunchKernelGGL(kv_check_finish_kernel, dim3(1), dim3(64), 0, stream, result);
  return hipGetLastError() == hipSuccess ? TOPKV_OK : TOPKV_ERR_LAUNCH;
}

}  // extern "C"
