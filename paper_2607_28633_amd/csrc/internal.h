// internal.h - calls between the library's own sources (not part of the C ABI).
#ifndef TOPKV_INTERNAL_H_
#define TOPKV_INTERNAL_H_

#include "topkv.h"

namespace topkv_internal {

// A plain pack (pool -> packed, every head) or unpack (packed -> pool) of one
// request with no window, run by the layout-move kernel's one-request direct
// grid when that grid applies (a token's pieces fill whole wave spans).  The
// length is the device value seq_lens[0], or seq_len (>= 0) when seq_lens is
// null.  *launched tells whether it launched; when it did not, nothing was
// queued and the caller launches its own kernel.  The caller has validated
// the arguments; `launch` carries the stream and the optional start/stop
// events.
__attribute__((visibility("hidden")))
topkv_status_t single_request_move(bool pack, const topkv_pool_t* pool, int32_t layer, void* packed,
                                   int64_t packed_cap, const int32_t* tables, int32_t bt_stride,
                                   const int32_t* seq_lens, int32_t seq_len, const topkv_launch_t* launch,
                                   bool* launched);

// One request with caller-placed planes, layers [first_layer, first_layer +
// layers) in one launch: plane c of layer first_layer + z is at packed +
// z * layer_stride + c * plane_stride, and the last byte moved must lie
// within packed_cap.  TOPKV_ERR_UNSUPPORTED (nothing queued) when one
// layer's work is too large for the direct grid that carries the layer
// dimension; the caller then moves the layers one launch each.
__attribute__((visibility("hidden")))
topkv_status_t placed_layers_move(bool pack, const topkv_pool_t* pool, int32_t first_layer, int32_t layers,
                                  void* packed, int64_t packed_cap, int64_t plane_stride, int64_t layer_stride,
                                  const int32_t* block_table, int32_t seq_len, hipStream_t stream);

// The pool descriptor checks every pack/unpack applies (positive sizes,
// element size 1/2/4/8, no overflow of the pool's byte size, row and page
// count within 32 bits): TOPKV_OK, or the status such a call would return.
__attribute__((visibility("hidden")))
topkv_status_t pool_ok(const topkv_pool_t* pool);

// Checked mode: true when the environment holds TOPKV_CHECKED=1 (read on
// every call, so it can be switched at run time).
__attribute__((visibility("hidden")))
bool checked_mode();

// Checked mode's validation of a pack/unpack call, run on `stream` before its
// launch, then synchronised: table entries of every page the move reads
// (within the window, when window > 0) in [0, num_pages), lengths in
// [0, bt_stride * page_size], with `duplicates` no destination page named
// twice, and the packed buffer large enough: fixed_bytes + per_token * (kept
// tokens of the batch) <= packed_cap.  The length is the device seq_lens[r],
// or seq_len for one request when seq_lens is null.  TOPKV_ERR_BOUNDS when
// anything fails (nothing is moved), TOPKV_ERR_UNSUPPORTED under stream
// capture.  Uses a per-device buffer the library allocates on first use.
__attribute__((visibility("hidden")))
topkv_status_t checked_tables(const topkv_pool_t* pool, int32_t num_reqs, const int32_t* block_tables,
                              int32_t bt_stride, const int32_t* seq_lens, int32_t seq_len, int32_t window,
                              bool duplicates, int64_t per_token, int64_t fixed_bytes, int64_t packed_cap,
                              hipStream_t stream);

// The same for a fixed-state layer: every slot in [0, num_slots), and with
// `duplicates` no slot named twice.
__attribute__((visibility("hidden")))
topkv_status_t checked_slots(const topkv_state_pool_t* pool, int32_t num_reqs, const int32_t* slots,
                             bool duplicates, hipStream_t stream);

}  // namespace topkv_internal

#endif  // TOPKV_INTERNAL_H_
