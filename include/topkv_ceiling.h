/*
 * topkv_ceiling.h - measurement kernels of libtopkv_ceiling.so (gfx950).
 *
 * Not part of the pack/unpack path: plain copies and an empty kernel that
 * give the practical ceiling and floor against which the pack / unpack
 * kernels of libtopkv.so are read.  The paper fixes the bytes a layer moves
 * (Section 2.2, Eq. 1: 2 * h_kv * d_h * s * b_p per layer); these kernels
 * move the same number of bytes with no block table at all, so the gap
 * between them and a pack or unpack is what the paging costs.  The copy
 * kernels use the pack/unpack kernels' copy core: 256-thread workgroups,
 * 8 x 16-byte vectors per lane (32 KiB per tile), every load of a tile
 * issued before its stores, non-temporal loads and stores.
 *
 * Plain device pointers and sizes; the caller owns all memory; nothing is
 * allocated or synchronised.  Errors: TOPKV_ERR_INVALID_ARG (topkv.h codes)
 * for null pointers, negative sizes, or pointers / sizes that are not
 * multiples of 16 bytes; TOPKV_ERR_LAUNCH when the runtime refuses the
 * launch; TOPKV_ERR_DEVICE when a device query fails.  Zero bytes launch
 * nothing.
 */
#ifndef TOPKV_CEILING_H_
#define TOPKV_CEILING_H_

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#include "topkv.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Copy `bytes` from src to dst in one launch, one 32 KiB tile per
 * workgroup (the per-layer launches' shape). */
topkv_status_t topkv_ceiling_copy(const void* src, void* dst, int64_t bytes, hipStream_t stream);

/* Copy `layers` blocks of layer_bytes (block z from src + z * src_stride to
 * dst + z * dst_stride) in ONE launch with the layer engine's schedule: a
 * persistent grid of workgroups_per_cu (0: 8) workgroups per compute unit
 * whose workgroup b copies tiles b, b + grid, ... of the layers in order.
 * The layer engine's transfer with contiguous pages and no table. */
topkv_status_t topkv_ceiling_copy_layers(const void* src, int64_t src_stride, void* dst, int64_t dst_stride,
                                         int64_t layer_bytes, int32_t layers, int32_t workgroups_per_cu,
                                         hipStream_t stream);

/* Read `bytes` at src, one 32 KiB tile per workgroup, and write the XOR of
 * tile b's 32-bit words to sink[b] (device memory, ceil(bytes / 32 KiB)
 * words): the read-only ceiling a checksum pass is read against. */
topkv_status_t topkv_ceiling_read(const void* src, int64_t bytes, uint32_t* sink, hipStream_t stream);

/* Copy `tiles` tiles in ONE launch, one workgroup per tile: tile k moves
 * lens[k] bytes (every tile 32 KiB when lens is null) from src + src_off[k]
 * to dst + dst_off[k] (src_off, dst_off: device int64 arrays of byte
 * offsets; lens: device int32 array or null).  A tile whose offsets or
 * length are not multiples of 16, whose length is not in [16, 32 KiB], or
 * whose bytes would leave [0, src_bytes) or [0, dst_bytes) is skipped.
 * With the offsets of a workload's page runs (the pages its block tables
 * name) this is the paged transfer with the table lookups and the length
 * arithmetic taken out: the ceiling of a pack or unpack over the same
 * scattered pages. */
topkv_status_t topkv_ceiling_copy_tiles(const void* src, int64_t src_bytes, const int64_t* src_off, void* dst,
                                        int64_t dst_bytes, const int64_t* dst_off, const int32_t* lens,
                                        int32_t tiles, hipStream_t stream);

/* One workgroup of 64 lanes that touches no memory: the cost of a launch. */
topkv_status_t topkv_ceiling_empty(hipStream_t stream);

/* As topkv_ceiling_copy, and workgroup b writes three wall-clock stamps to
 * stamps[3b .. 3b + 2] (device memory, ceil(bytes / 32 KiB) * 3 words):
 * when it starts, when its loads have returned, and when its stores have
 * completed.  The clock runs at topkv_ceiling_wall_clock_khz. */
topkv_status_t topkv_ceiling_copy_timeline(const void* src, void* dst, int64_t bytes, uint64_t* stamps,
                                           hipStream_t stream);

/* Frequency of the wall clock the stamps use, in kHz, for the current
 * device. */
topkv_status_t topkv_ceiling_wall_clock_khz(int32_t* khz);

#ifdef __cplusplus
}
#endif

#endif /* TOPKV_CEILING_H_ */
