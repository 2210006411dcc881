// state.hip - fixed-state layers (Section 2.2: a linear-attention layer holds,
// per request, a state whose size does not depend on the sequence length;
// Section 5.2: the unit of transfer is one layer).
//
// A serving engine keeps that state in a slot of a state cache laid out
// [layer][slot][state_bytes].  Packing a layer copies request r's state
// (slot slots[r]) to bytes [r * state_bytes, (r + 1) * state_bytes) of the
// packed buffer; unpacking is the inverse.  Every state is one contiguous run,
// so this is a streaming gather/scatter with no index math beyond one slot
// lookup per workgroup: a direct grid of (tile, request) workgroups, 256
// threads, up to 8 vectors of 16 bytes per lane (32 KiB tiles), all loads of
// a tile issued before its stores, non-temporal hints on full tiles.  Slots
// outside the cache are skipped, so bad device data cannot move bytes
// outside the two buffers.
#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>

#include <cstdint>

#include "internal.h"
#include "topkv.h"

#ifndef TOPKV_STATE_LDS_PAD
#define TOPKV_STATE_LDS_PAD 81920   // dynamic LDS bytes per workgroup for large states: 2 workgroups per CU
#endif

namespace topkv_state {

constexpr int kThreads = 256;
constexpr int kMaxVpt = 8;
constexpr int kMaxGridY = 65535;

template <int B> struct Vec;
template <> struct Vec<16> { typedef unsigned int type __attribute__((ext_vector_type(4))); };
template <> struct Vec<8> { typedef unsigned int type __attribute__((ext_vector_type(2))); };
template <> struct Vec<4> { typedef unsigned int type; };
template <> struct Vec<2> { typedef unsigned short type; };
template <> struct Vec<1> { typedef unsigned char type; };

struct StateParams {
  int64_t state_bytes;   // one request's state
  int64_t num_slots;     // valid slots are [0, num_slots)
  int64_t tile_bytes;    // kThreads * VPT * VB
  int32_t num_reqs;
  int32_t pad_;
};

// Copy `len` bytes (a multiple of VB, at most one tile) from src to dst:
// lane t handles vectors t, t + kThreads, ... so each wave instruction covers
// one contiguous 64-vector span.  A ragged tile clamps its load indices into
// the tile (loads stay unpredicated) and predicates only the stores.
template <int VB, int VPT>
__device__ __forceinline__ void copy_tile(char* __restrict__ dst, const char* __restrict__ src, int32_t len) {
  typedef typename Vec<VB>::type V;
  const V* __restrict__ s = reinterpret_cast<const V*>(src);
  V* __restrict__ d = reinterpret_cast<V*>(dst);
  const int32_t nv = len / VB;
  V v[VPT];
  if (nv == kThreads * VPT) {
#pragma unroll
    for (int j = 0; j < VPT; ++j) v[j] = __builtin_nontemporal_load(s + j * kThreads + threadIdx.x);
#pragma unroll
    for (int j = 0; j < VPT; ++j) __builtin_nontemporal_store(v[j], d + j * kThreads + threadIdx.x);
  } else {
#pragma unroll
    for (int j = 0; j < VPT; ++j) {
      const int idx = j * kThreads + (int)threadIdx.x;
      v[j] = s[idx < nv ? idx : nv - 1];
    }
#pragma unroll
    for (int j = 0; j < VPT; ++j) {
      const int idx = j * kThreads + (int)threadIdx.x;
      if (idx < nv) d[idx] = v[j];
    }
  }
}

// blockIdx.x = tile of a state, blockIdx.y = request (striding by gridDim.y
// when there are more requests than the grid's y extent).
template <int VB, int VPT, bool kPack>
__global__ __launch_bounds__(kThreads) void kv_state_kernel(char* __restrict__ layer_base,
                                                            char* __restrict__ packed,
                                                            const int32_t* __restrict__ slots, StateParams p) {
  const int64_t off = (int64_t)blockIdx.x * p.tile_bytes;
  const int64_t rem = p.state_bytes - off;
  const int32_t len = (int32_t)(rem < p.tile_bytes ? rem : p.tile_bytes);
  for (int32_t r = blockIdx.y; r < p.num_reqs; r += gridDim.y) {
    const int32_t slot = slots[r];
    if (slot < 0 || slot >= p.num_slots) continue;   // not a slot of this cache: skipped
    char* pool = layer_base + (int64_t)slot * p.state_bytes + off;
    char* pk = packed + (int64_t)r * p.state_bytes + off;
    if (kPack) copy_tile<VB, VPT>(pk, pool, len);
    else copy_tile<VB, VPT>(pool, pk, len);
  }
}

typedef void (*KernelFn)(char*, char*, const int32_t*, StateParams);

template <int VB, int VPT>
KernelFn kernel_for(bool pack) {
  return pack ? kv_state_kernel<VB, VPT, true> : kv_state_kernel<VB, VPT, false>;
}

KernelFn pick(bool pack, int vb, int vpt) {
  switch (vb) {
    case 16:
      switch (vpt) {
        case 8: return kernel_for<16, 8>(pack);
        case 4: return kernel_for<16, 4>(pack);
        case 2: return kernel_for<16, 2>(pack);
        default: return kernel_for<16, 1>(pack);
      }
    case 8: return kernel_for<8, kMaxVpt>(pack);
    case 4: return kernel_for<4, kMaxVpt>(pack);
    case 2: return kernel_for<2, kMaxVpt>(pack);
    default: return kernel_for<1, kMaxVpt>(pack);
  }
}

// Bytes of one layer of the cache, or -1 for a bad descriptor / overflow.
int64_t layer_bytes(const topkv_state_pool_t* pool) {
  if (!pool || !pool->base || pool->num_slots <= 0 || pool->state_bytes <= 0 || pool->num_layers <= 0 ||
      pool->reserved != 0)
    return -1;
  int64_t lay, all;
  if (__builtin_mul_overflow(pool->num_slots, pool->state_bytes, &lay) ||
      __builtin_mul_overflow(lay, (int64_t)pool->num_layers, &all))
    return -1;
  return lay;
}

topkv_status_t launch_state(bool pack, const topkv_state_pool_t* pool, int32_t layer, int32_t num_reqs,
                            const int32_t* slots, void* packed, int64_t packed_bytes,
                            const topkv_launch_t* launch) {
  const int64_t lay = layer_bytes(pool);
  if (lay < 0 || !launch) return TOPKV_ERR_INVALID_ARG;
  if (layer < 0 || layer >= pool->num_layers || num_reqs < 0 || packed_bytes < 0) return TOPKV_ERR_INVALID_ARG;
  if (num_reqs == 0) return TOPKV_OK;
  if (!slots || !packed) return TOPKV_ERR_INVALID_ARG;
  int64_t need;
  if (__builtin_mul_overflow((int64_t)num_reqs, pool->state_bytes, &need)) return TOPKV_ERR_UNSUPPORTED;
  if (packed_bytes < need) return TOPKV_ERR_INVALID_ARG;   // the batch must fit the packed buffer
  if (topkv_internal::checked_mode()) {
    const topkv_status_t st = topkv_internal::checked_slots(pool, num_reqs, slots, !pack, launch->stream);
    if (st != TOPKV_OK) return st;
  }

  char* base = static_cast<char*>(pool->base) + (int64_t)layer * lay;
  int vb = 16;
  while (vb > 1 && (reinterpret_cast<uintptr_t>(base) % vb || reinterpret_cast<uintptr_t>(packed) % vb ||
                    pool->state_bytes % vb))
    vb >>= 1;
  int vpt = kMaxVpt;
  if (vb == 16)   // smallest tile that still covers a small state in one pass
    while (vpt > 1 && (int64_t)kThreads * (vpt / 2) * vb >= pool->state_bytes) vpt >>= 1;
  StateParams p;
  p.state_bytes = pool->state_bytes;
  p.num_slots = pool->num_slots;
  p.tile_bytes = (int64_t)kThreads * vpt * vb;
  p.num_reqs = num_reqs;
  p.pad_ = 0;
  const int64_t tiles = (pool->state_bytes + p.tile_bytes - 1) / p.tile_bytes;
  if (tiles > INT32_MAX) return TOPKV_ERR_UNSUPPORTED;
  const dim3 grid((unsigned)tiles, (unsigned)(num_reqs < kMaxGridY ? num_reqs : kMaxGridY));
  char* pk = static_cast<char*>(packed);
  const KernelFn fn = pick(pack, vb, vpt);
  // Every workgroup of a large-state launch is live and moves a full 32 KiB
  // tile; two resident per CU (64 KiB in flight) beat eight by 2% on the
  // hybrid model's 2.2 MB states.  An LDS reservation the kernel never
  // touches sets that residency; small states keep full residency.
  const size_t lds = (vb == 16 && vpt == kMaxVpt && pool->state_bytes >= (1 << 20)) ? TOPKV_STATE_LDS_PAD : 0;
  if (launch->start || launch->stop)
    hipExtLaunchKernelGGL(fn, grid, dim3(kThreads), lds, launch->stream, launch->start, launch->stop, 0, base, pk,
                          slots, p);
  else
    hipLaunchKernelGGL(fn, grid, dim3(kThreads), lds, launch->stream, base, pk, slots, p);
  return hipGetLastError() == hipSuccess ? TOPKV_OK : TOPKV_ERR_LAUNCH;
}

}  // namespace topkv_state

extern "C" {

int64_t topkv_packed_state_bytes(const topkv_state_pool_t* pool, int32_t num_reqs) {
  if (topkv_state::layer_bytes(pool) < 0 || num_reqs < 0) return -1;
  int64_t b;
  if (__builtin_mul_overflow((int64_t)num_reqs, pool->state_bytes, &b)) return -1;
  return b;
}

topkv_status_t topkv_pack_state_layer(const topkv_state_pool_t* src, int32_t layer, int32_t num_reqs,
                                      const int32_t* slots, void* dst, int64_t dst_bytes,
                                      const topkv_launch_t* launch) {
  return topkv_state::launch_state(true, src, layer, num_reqs, slots, dst, dst_bytes, launch);
}

topkv_status_t topkv_unpack_state_layer(const void* src, int64_t src_bytes, const topkv_state_pool_t* dst,
                                        int32_t layer, int32_t num_reqs, const int32_t* slots,
                                        const topkv_launch_t* launch) {
  return topkv_state::launch_state(false, dst, layer, num_reqs, slots, const_cast<void*>(src), src_bytes, launch);
}

}  // extern "C"
