// ceiling.hip - measurement kernels (include/topkv_ceiling.h): plain copies
// with the pack/unpack kernels' copy core and an empty kernel, the ceiling
// and floor the pack / unpack kernels are read against.  Built as its own
// library; nothing on the pack/unpack path calls it.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "topkv_ceiling.h"

namespace topkv_ceiling {

constexpr int kThreads = 256;
constexpr int kVpt = 8;                                 // 16-byte vectors per lane per tile
constexpr int64_t kTile = (int64_t)kThreads * kVpt * 16;
typedef unsigned int V __attribute__((ext_vector_type(4)));

// Tile t of a copy of n16 16-byte vectors: lane j moves vectors
// t * 2048 + v * 256 + j, so each wave instruction covers one contiguous
// 1 KiB span; loads of a ragged last tile are clamped into the copy.
__device__ __forceinline__ void load_tile(V (&v)[kVpt], const V* __restrict__ s, int64_t base, int64_t n16) {
#pragma unroll
  for (int j = 0; j < kVpt; ++j) {
    const int64_t i = base + j * kThreads + threadIdx.x;
    v[j] = __builtin_nontemporal_load(s + (i < n16 ? i : n16 - 1));
  }
}

__device__ __forceinline__ void store_tile(const V (&v)[kVpt], V* __restrict__ d, int64_t base, int64_t n16) {
#pragma unroll
  for (int j = 0; j < kVpt; ++j) {
    const int64_t i = base + j * kThreads + threadIdx.x;
    if (i < n16) __builtin_nontemporal_store(v[j], d + i);
  }
}

__global__ __launch_bounds__(kThreads) void ceiling_copy_kernel(const V* __restrict__ s, V* __restrict__ d,
                                                                int64_t n16) {
  V v[kVpt];
  const int64_t base = (int64_t)blockIdx.x * kThreads * kVpt;
  load_tile(v, s, base, n16);
  store_tile(v, d, base, n16);
}

// tiles_per_layer tiles per layer, layers in order over a persistent grid
__global__ __launch_bounds__(kThreads) void ceiling_copy_layers_kernel(const char* __restrict__ src,
                                                                       int64_t src_stride, char* __restrict__ dst,
                                                                       int64_t dst_stride, int64_t layer16,
                                                                       int64_t tiles_per_layer, int64_t total) {
  for (int64_t w = blockIdx.x; w < total; w += gridDim.x) {
    const int64_t z = w / tiles_per_layer;
    const int64_t t = w - z * tiles_per_layer;
    V v[kVpt];
    const V* s = reinterpret_cast<const V*>(src + z * src_stride);
    V* d = reinterpret_cast<V*>(dst + z * dst_stride);
    load_tile(v, s, t * kThreads * kVpt, layer16);
    store_tile(v, d, t * kThreads * kVpt, layer16);
  }
}

// Read-only: each workgroup reads its 32 KiB tile and writes the XOR of it
// as one word to sink[blockIdx.x] (so the loads cannot be dropped).
__global__ __launch_bounds__(kThreads) void ceiling_read_kernel(const V* __restrict__ s, int64_t n16,
                                                                uint32_t* __restrict__ sink) {
  __shared__ uint32_t part[kThreads / 64];
  V v[kVpt];
  const int64_t base = (int64_t)blockIdx.x * kThreads * kVpt;
  load_tile(v, s, base, n16);
  uint32_t x = 0;
#pragma unroll
  for (int j = 0; j < kVpt; ++j)   // a ragged tile's clamped loads repeat its last vector: count it once
    if (base + j * kThreads + threadIdx.x < n16) x ^= v[j].x ^ v[j].y ^ v[j].z ^ v[j].w;
  for (int o = 32; o > 0; o >>= 1) x ^= __shfl_xor(x, o);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = x;
  __syncthreads();
  if (threadIdx.x == 0) sink[blockIdx.x] = part[0] ^ part[1] ^ part[2] ^ part[3];
}

// Tile w: lens[w] bytes (32 KiB when lens is null) from src + src_off[w] to dst + dst_off[w] (byte
// offsets); a tile whose offsets or length are not multiples of 16, whose length is not in
// [16, 32 KiB], or whose bytes would leave either buffer is skipped.
__global__ __launch_bounds__(kThreads) void ceiling_copy_tiles_kernel(const char* __restrict__ src, int64_t src_bytes,
                                                                      const int64_t* __restrict__ src_off,
                                                                      char* __restrict__ dst, int64_t dst_bytes,
                                                                      const int64_t* __restrict__ dst_off,
                                                                      const int32_t* __restrict__ lens) {
  const int64_t so = src_off[blockIdx.x], d0 = dst_off[blockIdx.x];
  const int64_t len = lens ? lens[blockIdx.x] : kTile;
  if (((so | d0 | len) & 15) || len < 16 || len > kTile || so < 0 || d0 < 0 || so > src_bytes - len ||
      d0 > dst_bytes - len)
    return;
  V v[kVpt];
  load_tile(v, reinterpret_cast<const V*>(src + so), 0, len / 16);
  store_tile(v, reinterpret_cast<V*>(dst + d0), 0, len / 16);
}

__global__ void ceiling_empty_kernel() {}

__global__ __launch_bounds__(kThreads) void ceiling_timeline_kernel(const V* __restrict__ s, V* __restrict__ d,
                                                                    int64_t n16, uint64_t* __restrict__ stamps) {
  const uint64_t t0 = (uint64_t)wall_clock64();
  V v[kVpt];
  const int64_t base = (int64_t)blockIdx.x * kThreads * kVpt;
  load_tile(v, s, base, n16);
  // the loads' data is needed before the clock is read again
  uint32_t sink = 0;
#pragma unroll
  for (int j = 0; j < kVpt; ++j) sink |= v[j].x;
  asm volatile("" ::"v"(sink));
  const uint64_t t1 = (uint64_t)wall_clock64();
  store_tile(v, d, base, n16);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // this wave's stores have completed
  __syncthreads();
  const uint64_t t2 = (uint64_t)wall_clock64();
  if (threadIdx.x == 0) {
    stamps[3 * blockIdx.x] = t0;
    stamps[3 * blockIdx.x + 1] = t1;
    stamps[3 * blockIdx.x + 2] = t2;
  }
}

bool aligned(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

topkv_status_t cu_count(int* out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return TOPKV_ERR_DEVICE;
  if (hipDeviceGetAttribute(out, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || *out <= 0)
    return TOPKV_ERR_DEVICE;
  return TOPKV_OK;
}

}  // namespace topkv_ceiling

extern "C" {

topkv_status_t topkv_ceiling_copy(const void* src, void* dst, int64_t bytes, hipStream_t stream) {
  using namespace topkv_ceiling;
  if (!src || !dst || bytes < 0 || bytes % 16 || !aligned(src) || !aligned(dst)) return TOPKV_ERR_INVALID_ARG;
  const int64_t tiles = (bytes + kTile - 1) / kTile;
  if (tiles == 0) return TOPKV_OK;
  if (tiles > INT32_MAX) return TOPKV_ERR_UNSUPPORTED;
  hipLaunchKernelGGL(ceiling_copy_kernel, dim3((unsigned)tiles), dim3(kThreads), 0, stream,
                     static_cast<const V*>(src), static_cast<V*>(dst), bytes / 16);
  return hipGetLastError() == hipSuccess ? TOPKV_OK : TOPKV_ERR_LAUNCH;
}

topkv_status_t topkv_ceiling_copy_layers(const void* src, int64_t src_stride, void* dst, int64_t dst_stride,
                                         int64_t layer_bytes, int32_t layers, int32_t workgroups_per_cu,
                                         hipStream_t stream) {
  using namespace topkv_ceiling;
  if (!src || !dst || layer_bytes < 0 || layer_bytes % 16 || layers < 0 || src_stride % 16 || dst_stride % 16 ||
      !aligned(src) || !aligned(dst) || workgroups_per_cu < 0 || workgroups_per_cu > 64)
    return TOPKV_ERR_INVALID_ARG;
  const int64_t tiles = (layer_bytes + kTile - 1) / kTile;
  if (tiles == 0 || layers == 0) return TOPKV_OK;
  int cus = 0;
  const topkv_status_t st = cu_count(&cus);
  if (st != TOPKV_OK) return st;
  const int64_t total = tiles * layers;
  const int64_t cap = (int64_t)cus * (workgroups_per_cu ? workgroups_per_cu : 8);
  hipLaunchKernelGGL(ceiling_copy_layers_kernel, dim3((unsigned)(total < cap ? total : cap)), dim3(kThreads), 0,
                     stream, static_cast<const char*>(src), src_stride, static_cast<char*>(dst), dst_stride,
                     layer_bytes / 16, tiles, total);
  return hipGetLastError() == hipSuccess ? TOPKV_OK : TOPKV_ERR_LAUNCH;
}

topkv_status_t topkv_ceiling_read(const void* src, int64_t bytes, uint32_t* sink, hipStream_t stream) {
  using namespace topkv_ceiling;
  if (!src || !sink || bytes < 0 || bytes % 16 || !aligned(src)) return TOPKV_ERR_INVALID_ARG;
  const int64_t tiles = (bytes + kTile - 1) / kTile;
  if (tiles == 0) return TOPKV_OK;
  if (tiles > INT32_MAX) return TOPKV_ERR_UNSUPPORTED;
  hipLaunchKernelGGL(ceiling_read_kernel, dim3((unsigned)tiles), dim3(kThreads), 0, stream,
                     static_cast<const V*>(src), bytes / 16, sink);
  return hipGetLastError() == hipSuccess ? TOPKV_OK : TOPKV_ERR_LAUNCH;
}

topkv_status_t topkv_ceiling_copy_tiles(const void* src, int64_t src_bytes, const int64_t* src_off, void* dst,
                                        int64_t dst_bytes, const int64_t* dst_off, const int32_t* lens,
                                        int32_t tiles, hipStream_t stream) {
  using namespace topkv_ceiling;
  if (!src || !dst || !src_off || !dst_off || src_bytes < 0 || dst_bytes < 0 || tiles < 0 || !aligned(src) ||
      !aligned(dst))
    return TOPKV_ERR_INVALID_ARG;
  if (tiles == 0) return TOPKV_OK;
  hipLaunchKernelGGL(ceiling_copy_tiles_kernel, dim3((unsigned)tiles), dim3(kThreads), 0, stream,
                     static_cast<const char*>(src), src_bytes, src_off, static_cast<char*>(dst), dst_bytes, dst_off,
                     lens);
  return hipGetLastError() == hipSuccess ? TOPKV_OK : TOPKV_ERR_LAUNCH;
}

topkv_status_t topkv_ceiling_empty(hipStream_t stream) {
  using namespace topkv_ceiling;
  hipLaunchKernelGGL(ceiling_empty_kernel, dim3(1), dim3(64), 0, stream);
  return hipGetLastError() == hipSuccess ? TOPKV_OK : TOPKV_ERR_LAUNCH;
}

topkv_status_t topkv_ceiling_copy_timeline(const void* src, void* dst, int64_t bytes, uint64_t* stamps,
                                           hipStream_t stream) {
  using namespace topkv_ceiling;
  if (!src || !dst || !stamps || bytes < 0 || bytes % 16 || !aligned(src) || !aligned(dst))
    return TOPKV_ERR_INVALID_ARG;
  const int64_t tiles = (bytes + kTile - 1) / kTile;
  if (tiles == 0) return TOPKV_OK;
  if (tiles > INT32_MAX) return TOPKV_ERR_UNSUPPORTED;
  hipLaunchKernelGGL(ceiling_timeline_kernel, dim3((unsigned)tiles), dim3(kThreads), 0, stream,
                     static_cast<const V*>(src), static_cast<V*>(dst), bytes / 16, stamps);
  return hipGetLastError() == hipSuccess ? TOPKV_OK : TOPKV_ERR_LAUNCH;
}

topkv_status_t topkv_ceiling_wall_clock_khz(int32_t* khz) {
  if (!khz) return TOPKV_ERR_INVALID_ARG;
  int dev = 0, v = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&v, hipDeviceAttributeWallClockRate, dev) != hipSuccess ||
      v <= 0)
    return TOPKV_ERR_DEVICE;
  *khz = v;
  return TOPKV_OK;
}

}  // extern "C"
