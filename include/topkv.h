/*
 * topkv.h - per-layer paged KV-cache pack / unpack for AMD MI355X (gfx950).
 *
 * C ABI of libtopkv.so.  Every entry point takes plain device pointers and
 * sizes, launches hand-written HIP kernels on the caller's stream and returns
 * without synchronising.  The library never allocates, frees or keeps
 * per-call state; it caches only each device's compute-unit count.  (Checked
 * mode, below, is the one exception: a debugging aid that allocates and
 * synchronises.)
 *
 * What is computed (arxiv 2607.28633, "Topology-Aware Data Movement for
 * Disaggregated GPU Inference"):
 *   - Section 5.2: a prefill worker sends layer l's KV cache while later
 *     layers still compute, so the unit of transfer is one layer.
 *   - Section 3.5: on the wire, K and V are contiguous tensors indexed
 *     [seq_len][kv_heads][head_dim] within a layer (single-DMA sends).
 *   - Section 6: both sides keep the cache in fixed-size pages reached
 *     through per-request block tables (PagedAttention).
 *   - Section 2.2, Eq. 1: a request of s tokens moves
 *     2 * L * h_kv * d_h * s * b_p bytes over L layers; Section 5.3: an MLA
 *     cache holds one shared latent per token and layer, no factor 2.
 *
 * Pool layout (topkv_pool_t), row-major:
 *     base[layer][page][plane][slot][head][dim]
 *   planes = 2 (K then V) or 1 (MLA latent); slot runs over page_size tokens;
 *   one element is elem_bytes opaque bytes (never interpreted: NaN payloads,
 *   -0 and subnormals are moved bit-exactly).  A "row" is one token of one
 *   plane: row_bytes = num_heads * head_dim * elem_bytes.
 *
 * Packed layout (one layer): per request r, in request order,
 *     [plane][token t < n_r][head][dim]
 *   so request r starts at byte planes * row_bytes * (n_0 + ... + n_{r-1}).
 *
 * Pack:   packed_r[c][t] = pool[layer][bt_r[t / P]][c][t % P]        t < n_r
 * Unpack: pool[layer][bt_r[t / P']][c][t % P'] = packed_r[c][t]      t < n_r
 *   where P / P' are the page sizes of the pool being read / written.  The
 *   packed form has no pages, so unpacking into a pool of another page size
 *   re-blocks.  Unpack writes only the slots of valid tokens: every other
 *   byte of the destination pool (other pages, and slots past the last token
 *   of a request's last page) keeps its value.
 *
 * Block tables: int32, device memory.  Entry i of request r is the physical
 * page (in [0, num_pages)) holding tokens [i*P, i*P + P).  Only the first
 * ceil(n_r / P) entries of a row are read; later entries may hold anything.
 * Within one unpack launch no destination page may be named twice (the
 * writes would race); pack has no such restriction.
 *
 * Errors: argument problems the host can see return a status before any
 * launch (TOPKV_ERR_INVALID_ARG for null pointers, out-of-range layer or
 * non-positive dimensions, TOPKV_ERR_UNSUPPORTED for sizes beyond the
 * documented limits).  A failed launch returns TOPKV_ERR_LAUNCH.  Device-side
 * contents are not trusted: a table entry outside [0, num_pages) makes the
 * kernel skip that page (nothing read or written for it); a device seq_len
 * below 0 counts as 0 and one above bt_stride * P as bt_stride * P; a batched
 * request whose packed block would cross the end of the packed buffer is not
 * moved.  Such skips are silent; topkv_check_tables reports bad entries and
 * lengths (and pages an unpack would write twice), and checked mode reports
 * all of them.  Overlapping source and destination ranges are undefined
 * behaviour.
 *
 * Checked mode: with TOPKV_CHECKED=1 in the environment (read on every
 * call), each pack / unpack call (every topkv_pack_layer* and
 * topkv_unpack_layer* call, and the KVCACHE1 layer calls) and each
 * fixed-state call first validates its device-side inputs on its stream,
 * synchronises that stream, and returns TOPKV_ERR_BOUNDS without moving
 * anything if a table entry the move would read lies outside [0, num_pages)
 * (with a window only the window's pages count), a length lies outside
 * [0, bt_stride * page_size], an unpack names a destination page twice, the
 * packed buffer cannot hold every kept token, or (fixed-state calls) a slot
 * lies outside the cache or an unpack names it twice.  A stream under
 * capture gets TOPKV_ERR_UNSUPPORTED (checked mode synchronises).  The
 * library allocates a small per-device buffer (16 bytes plus one bit per
 * pool page or state slot) on first use and keeps it until the process ends.
 *
 * Build: hipcc --offload-arch=gfx950 (see the package's build script).  C
 * callers compile with -D__HIP_PLATFORM_AMD__ -I/opt/rocm/include.
 */
#ifndef TOPKV_H_
#define TOPKV_H_

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum topkv_status {
  TOPKV_OK = 0,
  TOPKV_ERR_INVALID_ARG = 1,  /* null pointer, bad layer index, non-positive dimension */
  TOPKV_ERR_UNSUPPORTED = 2,  /* valid but beyond the library's limits (see each call) */
  TOPKV_ERR_LAUNCH = 3,       /* the HIP runtime refused the launch */
  TOPKV_ERR_BOUNDS = 4,       /* invalid device-side table, length, slot or capacity (checked path) */
  TOPKV_ERR_DEVICE = 5,       /* a HIP runtime query failed */
  TOPKV_ERR_CHECKSUM = 6,     /* topkv_kvcache1_verify: header or checksum mismatch */
  TOPKV_ERR_TIMEOUT = 7,      /* layer engine: a layer's ready word did not arrive in time (device status) */
  TOPKV_ERR_CANCELLED = 8     /* layer engine: the cancel word was set while a layer was awaited (device status) */
} topkv_status_t;

/* One paged KV pool.  The caller owns the memory.  All counts are elements
 * or tokens; layer stride = num_pages * planes * page_size * row_bytes. */
typedef struct topkv_pool {
  void*   base;        /* device pointer to base[num_layers][num_pages][planes][page_size][heads][dim] */
  int64_t num_pages;   /* pages per layer, > 0 */
  int32_t num_layers;  /* > 0 */
  int32_t page_size;   /* tokens per page, > 0 */
  int32_t planes;      /* 2 = K|V, 1 = MLA latent (any value > 0 is accepted) */
  int32_t num_heads;   /* KV heads, > 0 */
  int32_t head_dim;    /* > 0 */
  int32_t elem_bytes;  /* 1, 2, 4 or 8 (bf16/fp16 caches: 2) */
} topkv_pool_t;

/* Launch options for the *_ex calls.  When start / stop are non-null they
 * are stamped with the kernel's own begin / end time (hipExtLaunchKernel), so
 * hipEventElapsedTime(start, stop) is the kernel duration without queueing
 * gaps.  Events must have been created by the caller on the same device. */
typedef struct topkv_launch {
  hipStream_t stream;
  hipEvent_t  start;
  hipEvent_t  stop;
} topkv_launch_t;

/* Largest num_reqs one batched launch accepts (per-request prefix sums live
 * in LDS: 12 bytes per request).  Larger batches: split into launches.  A
 * launch's token capacity, num_reqs * bt_stride * page_size, must also stay
 * below 2^31 (TOPKV_ERR_UNSUPPORTED otherwise). */
#define TOPKV_MAX_BATCH_REQS 4096

/* Pack one request's tokens of one layer (Sections 5.2, 3.5, 6).
 *   src:         pool to read (device memory described by *src, host struct)
 *   layer:       in [0, src->num_layers)
 *   block_table: device int32[ceil(seq_len / src->page_size)]
 *   seq_len:     tokens, >= 0 (0: nothing is launched)
 *   dst:         device buffer of planes * seq_len * row_bytes bytes,
 *                written as [plane][seq_len][heads][dim]
 *   stream:      HIP stream the kernel is queued on */
topkv_status_t topkv_pack_layer(const topkv_pool_t* src, int32_t layer,
                                const int32_t* block_table, int32_t seq_len,
                                void* dst, hipStream_t stream);

/* Unpack one request's packed layer into a pool (inverse of
 * topkv_pack_layer; dst->page_size may differ from the page size the data
 * was packed from).  src holds planes * seq_len * row_bytes bytes. */
topkv_status_t topkv_unpack_layer(const void* src, const topkv_pool_t* dst, int32_t layer,
                                  const int32_t* block_table, int32_t seq_len,
                                  hipStream_t stream);

/* Pack num_reqs requests of one layer in ONE launch (Section 5.2 per-layer
 * unit; batching keeps small layers from being launch-bound).
 *   block_tables: device int32[num_reqs][bt_stride], bt_stride >= the
 *                 largest ceil(seq_lens[r] / page_size)
 *   seq_lens:     device int32[num_reqs]; request offsets in the packed
 *                 buffer are prefix sums computed on the device
 *   dst:          device buffer of dst_bytes bytes; the batch occupies the
 *                 first planes * row_bytes * sum(seq_lens) bytes
 *   num_reqs:     0 .. TOPKV_MAX_BATCH_REQS (0: nothing is launched) */
topkv_status_t topkv_pack_layer_batched(const topkv_pool_t* src, int32_t layer,
                                        int32_t num_reqs, const int32_t* block_tables,
                                        int32_t bt_stride, const int32_t* seq_lens,
                                        void* dst, int64_t dst_bytes, hipStream_t stream);

/* Unpack num_reqs packed requests of one layer in one launch (inverse of
 * topkv_pack_layer_batched; re-blocks when the pool's page size differs from
 * the packing side's).  src holds src_bytes bytes of packed data. */
topkv_status_t topkv_unpack_layer_batched(const void* src, int64_t src_bytes,
                                          const topkv_pool_t* dst, int32_t layer,
                                          int32_t num_reqs, const int32_t* block_tables,
                                          int32_t bt_stride, const int32_t* seq_lens,
                                          hipStream_t stream);

/* The batched calls with launch options (kernel-timestamp events).
 * launch must be non-null. */
topkv_status_t topkv_pack_layer_batched_ex(const topkv_pool_t* src, int32_t layer,
                                           int32_t num_reqs, const int32_t* block_tables,
                                           int32_t bt_stride, const int32_t* seq_lens,
                                           void* dst, int64_t dst_bytes,
                                           const topkv_launch_t* launch);
topkv_status_t topkv_unpack_layer_batched_ex(const void* src, int64_t src_bytes,
                                             const topkv_pool_t* dst, int32_t layer,
                                             int32_t num_reqs, const int32_t* block_tables,
                                             int32_t bt_stride, const int32_t* seq_lens,
                                             const topkv_launch_t* launch);

/* Layer engine (Section 5.2: a prefill worker sends layer l while layers
 * l+1 .. L-1 are still being computed, so the unit of transfer is one
 * layer).  ONE launch moves layers [first_layer, first_layer +
 * num_layers) of a batch, each layer exactly as topkv_pack_layer_batched /
 * topkv_unpack_layer_batched would move it, in layer order, and each layer
 * only once its ready word allows.  The per-launch costs of one launch per
 * layer (dispatch, the first table and length loads, each kernel's drain)
 * are paid once per range.  The tables and lengths are shared by every layer
 * of the range (one block table per request indexes every layer's pool).
 *   layer z of the range (pool layer first_layer + z) uses the packed block
 *   at packed + z * layer_stride, of min(layer_stride, packed_bytes -
 *   z * layer_stride) bytes (packed_bytes when num_layers == 1); a request
 *   whose packed block would cross that end is not moved in that layer, as
 *   in the batched calls.  layer_stride > 0 when num_layers > 1, and
 *   (num_layers - 1) * layer_stride <= packed_bytes.  Windowed and fixed-
 *   state layers use their own per-layer calls.
 *
 * Waiting (engine->ready non-null): ready[z] has reached the epoch when
 * (int32_t)(ready[z] - engine->epoch) >= 0, so the same words serve
 * successive transfers with increasing epochs; layers move in order, so
 * layer z may move once ready[0..z] have all reached it.  The words may
 * sit in device memory or in host memory the device can reach (pinned,
 * mapped); a producer publishes layer z by storing ready[z] with release
 * ordering after the layer's data (a host store after the data's copy has
 * completed, a kernel's release store, or a stream-ordered write after the
 * producing kernel).  Each wait is bounded: after engine->timeout_us
 * microseconds without the word, or as soon as the cancel word (optional,
 * device or host memory) is non-zero, the waiting workgroups give up and
 * exit: the layers before the first word that did not arrive are moved in
 * full, that layer and every later one are not touched.  The first reason
 * (TOPKV_ERR_TIMEOUT or TOPKV_ERR_CANCELLED) is written to *engine->status
 * (device int32 that must hold 0 at launch; it stays 0 when every layer
 * moved).  The status is written by the kernel: read it after the stream
 * has completed.  engine == NULL, or engine->ready == NULL: every layer
 * moves at once.
 *
 * Grids: without waiting, the launch is a hardware-dispatched grid with one
 * workgroup per (layer, request, table entry, plane, tile) slot, as the
 * batched calls use for one layer (slots past a request's pages exit at
 * once), issued as consecutive grids of topkv_engine_layers_per_grid layers
 * each (engine->layers_per_grid when non-zero, else about 512 MiB of packed
 * blocks per grid: a single grid over a long range was measured slower on
 * MI355X); beyond that grid's limits (more than 1024 requests, 2^20 slots per
 * layer, 65535 table entries or 65535 requests * layers) and whenever it
 * waits, the engine is a persistent grid that keeps
 * engine->workgroups_per_cu workgroups of 256 threads per compute unit (0: 8)
 * for the whole launch, each working through its share of the items in
 * layer order; a caller whose producer kernels must run beside a waiting
 * engine on the same GPU leaves them room with a smaller value (e.g. 2).
 * Returns synchronously: the host-
 * side argument errors of the batched calls, TOPKV_ERR_INVALID_ARG for a bad
 * layer range or layer_stride, a null status with ready set, or a timeout
 * outside (0, 60 000 000] us or a negative layers_per_grid, and
 * TOPKV_ERR_UNSUPPORTED when num_layers *
 * num_reqs * bt_stride * (items per page) reaches 2^31.  Checked mode
 * validates the tables and lengths once for the range (the smallest layer
 * block as capacity).  The call never synchronises otherwise and allocates
 * nothing. */
typedef struct topkv_engine {
  const uint32_t* ready;      /* [num_layers] words, or NULL (no waiting) */
  const uint32_t* cancel;     /* optional word; non-zero: waiting workgroups give up */
  int32_t*        status;     /* device int32, 0 at launch; required with ready */
  uint32_t        epoch;      /* value each ready word must reach */
  int32_t         workgroups_per_cu;  /* 0: 8 */
  int64_t         timeout_us; /* longest wait for one layer, in (0, 60e6]; ignored without ready */
  int32_t         layers_per_grid;    /* without ready: layers per hardware-dispatched grid, 0: the library's */
} topkv_engine_t;

/* Layers that each hardware-dispatched grid of an engine call without
 * waiting covers (the call's last grid may cover fewer): engine->
 * layers_per_grid when engine is non-null and it is non-zero (at most
 * num_layers), else num_layers cut into ceil(num_layers * layer_stride /
 * 512 MiB) grids of equal layer count, rounded up.  Host-only, no device
 * access; the persistent grid (waiting, or a range past the direct grid's
 * limits) is always one launch.  Returns -1 for num_layers < 1, a negative
 * layer_stride or a negative engine->layers_per_grid. */
int32_t topkv_engine_layers_per_grid(int32_t num_layers, int64_t layer_stride, const topkv_engine_t* engine);

topkv_status_t topkv_engine_pack_layers(const topkv_pool_t* src, int32_t first_layer, int32_t num_layers,
                                        int32_t num_reqs, const int32_t* block_tables, int32_t bt_stride,
                                        const int32_t* seq_lens, void* packed, int64_t layer_stride,
                                        int64_t packed_bytes, const topkv_engine_t* engine,
                                        hipStream_t stream);
topkv_status_t topkv_engine_unpack_layers(const void* packed, int64_t layer_stride, int64_t packed_bytes,
                                          const topkv_pool_t* dst, int32_t first_layer, int32_t num_layers,
                                          int32_t num_reqs, const int32_t* block_tables, int32_t bt_stride,
                                          const int32_t* seq_lens, const topkv_engine_t* engine,
                                          hipStream_t stream);

/* Windowed layers (Section 2.2 extends Eq. 1 per layer kind: a sliding-
 * window attention layer holds only its last `window` tokens).  As the
 * batched calls, but only tokens [max(0, n_r - window), n_r) of request r
 * move; window 0 moves every token (identical to the batched calls).  The
 * packed block of request r is [planes][min(n_r, window)][heads][dim];
 * unpack writes those tokens at their own positions t (page t / P', slot
 * t % P') and nothing else.  window < 0 is TOPKV_ERR_INVALID_ARG.
 * launch must be non-null. */
topkv_status_t topkv_pack_layer_window(const topkv_pool_t* src, int32_t layer, int32_t num_reqs,
                                       const int32_t* block_tables, int32_t bt_stride,
                                       const int32_t* seq_lens, int32_t window, void* dst,
                                       int64_t dst_bytes, const topkv_launch_t* launch);
topkv_status_t topkv_unpack_layer_window(const void* src, int64_t src_bytes,
                                         const topkv_pool_t* dst, int32_t layer, int32_t num_reqs,
                                         const int32_t* block_tables, int32_t bt_stride,
                                         const int32_t* seq_lens, int32_t window,
                                         const topkv_launch_t* launch);

/* Bytes of one layer's packed batch, planes * row_bytes * sum(seq_lens),
 * computed on the host from HOST seq_lens (Eq. 1 for one layer; planes = 1
 * for MLA per Section 5.3).  Returns -1 for a null/invalid pool, a null
 * seq_lens with num_reqs > 0, a negative length or int64 overflow. */
int64_t topkv_packed_layer_bytes(const topkv_pool_t* pool, const int32_t* seq_lens_host,
                                 int32_t num_reqs);

/* The same for a windowed layer: planes * row_bytes * sum(min(n_r, window))
 * (window 0: every token).  -1 also for window < 0. */
int64_t topkv_packed_window_bytes(const topkv_pool_t* pool, const int32_t* seq_lens_host,
                                  int32_t num_reqs, int32_t window);

/* One request with caller-placed planes: plane c of the packed request
 * (c < planes) is written to / read from dst + c * plane_stride as
 * [n][heads][dim] rows (plane_stride > 0; 16-byte multiples keep the wide
 * path).  With plane_stride = tensor bytes this writes one layer's K and V
 * rows straight into the K and V tensors of a serialized request
 * (Section 3.5).  dst_bytes / src_bytes: bytes available from dst / src;
 * the last plane must end within it, or nothing is moved. */
topkv_status_t topkv_pack_layer_planes(const topkv_pool_t* src, int32_t layer,
                                       const int32_t* block_table, int32_t seq_len, void* dst,
                                       int64_t plane_stride, int64_t dst_bytes, hipStream_t stream);
topkv_status_t topkv_unpack_layer_planes(const void* src, int64_t plane_stride, int64_t src_bytes,
                                         const topkv_pool_t* dst, int32_t layer,
                                         const int32_t* block_table, int32_t seq_len,
                                         hipStream_t stream);

/* ---- Whole-request serialization: KVCACHE1 (Section 3.5) --------------------
 * A blob is a 128-byte header followed by the K tensor and the V tensor,
 * each [layers][seq_len][kv_heads][head_dim] (the V tensor is empty for an
 * MLA cache, planes = 1, Section 5.3).  The paper fixes the fields but not
 * their widths, byte order or the CRC; this library writes, little-endian:
 *   0 "KVCACHE1"   8 request_id u64   16 model_id u64
 *   24 seq_len u32 28 layers u32      32 kv_heads u32   36 head_dim u32
 *   40 elem_bytes u32                 44 planes u32
 *   48 k_bytes u64 56 v_bytes u64     64 crc64(K) u64   72 crc64(V) u64
 *   80..127 zero
 * CRC-64/XZ: ECMA-182 polynomial 0x42F0E1EBA9EA3693, reflected, preset and
 * final complement all ones (CRC of "123456789" = 0x995DC9BBDF1939FA).
 * The pool descriptor gives the geometry (all num_layers layers go in the
 * blob); rows must be a multiple of 16 bytes and the blob 16-byte aligned
 * (TOPKV_ERR_UNSUPPORTED otherwise).  Typical sender: topkv_kvcache1_pack_
 * layer for each layer as it is produced, then topkv_kvcache1_seal; receiver:
 * topkv_kvcache1_verify, then topkv_kvcache1_unpack_layer per layer. */

/* Blob bytes for seq_len tokens (128 + planes * layers * seq_len * row); -1
 * for bad geometry. */
int64_t topkv_kvcache1_bytes(const topkv_pool_t* geometry, int32_t seq_len);

/* Workspace bytes seal / verify need (checksum partials); -1 on bad input. */
int64_t topkv_kvcache1_workspace_bytes(const topkv_pool_t* geometry, int32_t seq_len);

/* Pack layer `layer` of one request into its rows of the blob's K and V
 * tensors (one launch; block_table as for topkv_pack_layer). */
topkv_status_t topkv_kvcache1_pack_layer(const topkv_pool_t* src, int32_t layer,
                                         const int32_t* block_table, int32_t seq_len, void* blob,
                                         int64_t blob_bytes, hipStream_t stream);

/* Layers [first_layer, first_layer + num_layers) of one request packed into
 * their rows of the blob's K and V tensors in a few launches (a whole request
 * at once, when it is not shipped layer by layer): grids of
 * topkv_engine_layers_per_grid(num_layers, planes * seq_len * row bytes)
 * layers each, as the layer engine issues them; when one layer's work is too
 * large for such a grid, one launch per layer.  The same result as
 * topkv_kvcache1_pack_layer for each layer.  TOPKV_ERR_INVALID_ARG for a
 * layer range outside [0, src->num_layers), otherwise as
 * topkv_kvcache1_pack_layer; num_layers == 0 queues nothing. */
topkv_status_t topkv_kvcache1_pack_layers(const topkv_pool_t* src, int32_t first_layer, int32_t num_layers,
                                          const int32_t* block_table, int32_t seq_len, void* blob,
                                          int64_t blob_bytes, hipStream_t stream);

/* After every layer is packed: checksum both tensors on the device and write
 * the header.  workspace: topkv_kvcache1_workspace_bytes() bytes of device
 * memory owned by the caller (contents on return are scratch).  Queued on
 * stream; the blob is complete once the stream reaches this point. */
topkv_status_t topkv_kvcache1_seal(const topkv_pool_t* geometry, int32_t seq_len,
                                   uint64_t request_id, uint64_t model_id, void* blob,
                                   int64_t blob_bytes, void* workspace, int64_t workspace_bytes,
                                   hipStream_t stream);

/* Receiver check: recompute both checksums and compare them, and the header
 * fields, with what the caller expects.  result: device int32[4] written on
 * the stream: [0] TOPKV_OK or TOPKV_ERR_CHECKSUM, [1] bit mask of header
 * words 0-7 that differ, [2] K checksum mismatch, [3] V checksum mismatch.
 * A mismatch is the paper's trigger for a retry. */
topkv_status_t topkv_kvcache1_verify(const topkv_pool_t* geometry, int32_t seq_len,
                                     uint64_t request_id, uint64_t model_id, const void* blob,
                                     int64_t blob_bytes, void* workspace, int64_t workspace_bytes,
                                     int32_t* result, hipStream_t stream);

/* Scatter layer `layer` of a blob into a pool (any page size; the blob's
 * geometry is the pool descriptor's, seq_len tokens). */
topkv_status_t topkv_kvcache1_unpack_layer(const void* blob, int64_t blob_bytes,
                                           const topkv_pool_t* dst, int32_t layer,
                                           const int32_t* block_table, int32_t seq_len,
                                           hipStream_t stream);

/* Layers [first_layer, first_layer + num_layers) of a blob scattered into a
 * pool, in the same grids (see topkv_kvcache1_pack_layers). */
topkv_status_t topkv_kvcache1_unpack_layers(const void* blob, int64_t blob_bytes, const topkv_pool_t* dst,
                                            int32_t first_layer, int32_t num_layers, const int32_t* block_table,
                                            int32_t seq_len, hipStream_t stream);

/* Whole-request serialization in one pass (Section 3.5): every layer's K and
 * V rows move from the pool into the blob inside the CRC kernels that
 * checksum them, then the header is written.  The blob (header included) is
 * byte for byte what topkv_kvcache1_pack_layers(all layers) followed by
 * topkv_kvcache1_seal writes, including where a table entry lies outside the
 * pool (those rows keep the blob's bytes and are checksummed as they are);
 * the pool is read once and the blob written once instead of being written
 * and read back.  Same arguments and workspace as those two calls;
 * block_table: device int32[ceil(seq_len / page_size)].  Requests beyond the
 * one-pass limits (layers * seq_len >= 2^31, rows of 2^31 - 2^17 bytes or
 * more, a pool base off 16-byte alignment) take the two calls internally. */
topkv_status_t topkv_kvcache1_pack_seal(const topkv_pool_t* src, const int32_t* block_table,
                                        int32_t seq_len, uint64_t request_id, uint64_t model_id,
                                        void* blob, int64_t blob_bytes, void* workspace,
                                        int64_t workspace_bytes, hipStream_t stream);

/* Receiver in one pass: the blob's K and V tensors are checksummed and, in the
 * same kernels, scattered into every layer of the pool (any page size), and
 * the header is compared as topkv_kvcache1_verify does (same result words).
 * The pool pages named by block_table are written whatever the verdict: a
 * caller that sees result[0] != TOPKV_OK must treat them as garbage (and
 * retry the transfer).  Rows whose table entry lies outside the pool are not
 * written.  Same fallback limits as topkv_kvcache1_pack_seal. */
topkv_status_t topkv_kvcache1_verify_unpack(const void* blob, int64_t blob_bytes,
                                            const topkv_pool_t* dst, const int32_t* block_table,
                                            int32_t seq_len, uint64_t request_id, uint64_t model_id,
                                            void* workspace, int64_t workspace_bytes, int32_t* result,
                                            hipStream_t stream);

/* CRC-64/XZ (as above) of nbytes of device memory at data (16-byte aligned,
 * any length up to 256 spans of 2 GiB - 64 KiB, about 512 GiB, beyond any
 * one device's memory: TOPKV_ERR_UNSUPPORTED above that), written to the
 * device word *crc_out on the stream.
 * workspace: topkv_crc64_workspace_bytes(nbytes) bytes of device memory,
 * 8-byte aligned, caller-owned. */
topkv_status_t topkv_crc64(const void* data, int64_t nbytes, void* workspace,
                           int64_t workspace_bytes, uint64_t* crc_out, hipStream_t stream);
int64_t topkv_crc64_workspace_bytes(int64_t nbytes);

/* topkv_crc64 for callers that cannot allocate (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): no
 * workspace argument, and nothing is allocated or freed.  The workspace is a
 * file-scope device array of TOPKV_CRC64_NOALLOC_SCRATCH_BYTES bytes (at most
 * 256 span registers), one copy per GPU the library runs
 * on, held until the process ends; the first call on a device looks its
 * address up (hipGetSymbolAddress, device current), so make that call before
 * any capture on that device.  Every length fits that
 * array, so no length is refused for room; a length that needed more would
 * get TOPKV_ERR_UNSUPPORTED.  Same result, alignment rule (data 16-byte
 * aligned: TOPKV_ERR_UNSUPPORTED otherwise) and errors as topkv_crc64.
 * Calls on one GPU share its array: calls whose kernels overlap in time
 * (other streams, other threads) race and may write wrong checksums; calls
 * ordered on one stream are safe (each rewrites every word it reads). */
#define TOPKV_CRC64_NOALLOC_SCRATCH_BYTES 2048
topkv_status_t topkv_crc64_noalloc(const void* data, int64_t nbytes, uint64_t* crc_out,
                                   hipStream_t stream);

/* Checked path: validate block tables and lengths on the device before a
 * pack or unpack (the movement calls skip bad entries silently).  For every
 * request r and entry i < ceil(seq_lens[r] / pool->page_size) it checks
 * 0 <= entry < pool->num_pages, that seq_lens[r] lies in
 * [0, bt_stride * page_size], and, when check_duplicates != 0, that no page
 * is named twice in the batch (required of an unpack destination, where two
 * writers of one page would race; a pack source may repeat pages).
 *   pool:       geometry only (num_pages, page_size); base is not accessed
 *   workspace:  device memory of topkv_check_workspace_bytes(pool) bytes (a
 *               page bitmap), owned by the caller, cleared by this call; may
 *               be null when check_duplicates == 0
 *   result:     device int32[4], written on the stream: [0] TOPKV_OK or
 *               TOPKV_ERR_BOUNDS, [1] entries out of range, [2] repeated
 *               pages, [3] lengths out of range.  Read it after the stream
 *               has synchronised.
 * Launches three small kernels; the call itself does not synchronise.
 * Calls sharing a workspace on overlapping streams race. */
topkv_status_t topkv_check_tables(const topkv_pool_t* pool, int32_t num_reqs,
                                  const int32_t* block_tables, int32_t bt_stride,
                                  const int32_t* seq_lens, int32_t check_duplicates,
                                  void* workspace, int64_t workspace_bytes,
                                  int32_t* result, hipStream_t stream);

/* Workspace bytes topkv_check_tables needs for this pool (a bitmap of
 * num_pages bits, in 4-byte words); -1 for a null or empty pool. */
int64_t topkv_check_workspace_bytes(const topkv_pool_t* pool);

/* Layer moves between cache layouts (one layer, a batch of requests).
 *
 * A view is one side of a move:
 *   TOPKV_LAYOUT_PACKED           `data`/`bytes`: per request a block
 *                                 [planes][kept tokens][head_count][head_dim],
 *                                 blocks in request order (the pack/unpack
 *                                 wire order, restricted to the moved heads).
 *                                 With `shards` = S > 1 (tensor-parallel
 *                                 receivers) the moved heads split into S equal
 *                                 runs and shard s is such a buffer of its
 *                                 head_count / S heads at data + s * bytes
 *                                 (`bytes` is then each shard's capacity)
 *   TOPKV_LAYOUT_POOL             `pool`: the slot-major pool of topkv_pool_t,
 *                                 [layer][page][plane][slot][head][dim]
 *   TOPKV_LAYOUT_POOL_HEAD_MAJOR  `pool` geometry, but each page plane is
 *                                 [head][slot][dim] (each head's slots adjacent)
 * Pool views also give `layer`, `block_tables` (device int32
 * [num_reqs][bt_stride]) and `head_begin`, the first of the head_count moved
 * heads, and ignore `shards`.  Packed views ignore the pool fields; shards 0
 * or 1 means one region.
 *
 * For every request r, kept token t (the last `window` tokens when window > 0,
 * Sec. 2.2; all of them when 0), plane c, j < head_count and dim d:
 *   dst(r, t, c, dst.head_begin + j, d) = src(r, t, c, src.head_begin + j, d).
 * Token t of a pool view is page block_tables[r][t / page_size], slot
 * t % page_size of that pool (Sec. 6).  Nothing else in a destination pool is
 * written.  Cases: head-sliced pack (pool -> packed, the heads of one
 * tensor-parallel shard), head-sliced unpack (packed -> pool), re-blocking
 * between page sizes with no staging buffer (pool -> pool), and head-major
 * pools on either side.
 *
 * Requirements: at least one side is a pool; a packed side's shards divide
 * head_count (and, if S > 1, its piece width divides `bytes`); pool sides agree on planes,
 * head_dim and elem_bytes (page size, page count, head count and layer count
 * may differ); 1 <= head_count <= num_heads - head_begin on each pool side;
 * 0 <= num_reqs <= TOPKV_MAX_BATCH_REQS; seq_lens is device int32 [num_reqs].
 * Lengths are clamped on the device to [0, min over pool sides of
 * bt_stride * page_size]; entries outside [0, num_pages) are skipped, and so
 * are packed pieces past `bytes`.  src and dst must not overlap.
 * Errors: TOPKV_ERR_INVALID_ARG for bad descriptors or arguments,
 * TOPKV_ERR_UNSUPPORTED when a launch would address 2^31 or more pieces
 * (num_reqs * max tokens * planes * head_count * head_dim * elem_bytes / piece
 * width), TOPKV_ERR_LAUNCH if the launch fails.  One kernel on the stream;
 * the call does not synchronise. */
typedef enum topkv_layout {
    TOPKV_LAYOUT_PACKED = 0,
    TOPKV_LAYOUT_POOL = 1,
    TOPKV_LAYOUT_POOL_HEAD_MAJOR = 2
} topkv_layout_t;

typedef struct topkv_view {
    int32_t layout;               /* topkv_layout_t */
    int32_t layer;                /* pool views: layer index */
    int32_t head_begin;           /* pool views: first moved head */
    int32_t bt_stride;            /* pool views: entries per block-table row */
    const int32_t* block_tables;  /* pool views: device [num_reqs][bt_stride] */
    topkv_pool_t pool;            /* pool views: geometry and base */
    void* data;                   /* packed views: device buffer */
    int64_t bytes;                /* packed views: capacity in bytes (of each shard) */
    int32_t shards;               /* packed views: 0 or 1 = one region, S > 1 = S shard regions */
    int32_t reserved;             /* set to 0 */
} topkv_view_t;

topkv_status_t topkv_move_layer(const topkv_view_t* src, const topkv_view_t* dst, int32_t num_reqs,
                                const int32_t* seq_lens, int32_t head_count, int32_t window,
                                hipStream_t stream);

/* A range of layers moved as topkv_move_layer moves one (same views, rules
 * and errors), in a few launches instead of one per layer (a whole request
 * resharded, re-blocked or re-laid out at once, when it is not moved layer
 * by layer as the layers are produced, Section 5.2).  Layer z < num_layers
 * of a pool view is pool layer view.layer + z (so view.layer + num_layers
 * <= pool.num_layers); layer z of a packed view starts at data +
 * z * packed_layer_stride and holds that view's region(s) (`bytes`, or S
 * shard regions of `bytes` each), so with num_layers > 1 the stride is at
 * least max(1, shards) * bytes and the buffer spans (num_layers - 1) *
 * packed_layer_stride plus one layer's regions.  The layers go out as
 * hardware-dispatched grids of topkv_engine_layers_per_grid layers (the
 * bytes of one layer's packed regions, or for pool to pool the source
 * tables' capacity) where a direct grid applies (no window, whole wave
 * spans per token), else one launch per layer.  num_layers == 0 or
 * num_reqs == 0 queues nothing.  Extra errors: TOPKV_ERR_INVALID_ARG for a
 * negative num_layers or stride, a layer range outside a pool, or a stride
 * that would overlap consecutive layers' packed regions. */
topkv_status_t topkv_move_layers(const topkv_view_t* src, const topkv_view_t* dst, int32_t num_layers,
                                 int64_t packed_layer_stride, int32_t num_reqs, const int32_t* seq_lens,
                                 int32_t head_count, int32_t window, hipStream_t stream);

/* Head-sliced pack: heads [head_begin, head_begin + head_count) of layer
 * `layer` of a slot-major pool into dst ([planes][n_r][head_count][dim] per
 * request, requests concatenated; dst_bytes is its capacity).  Same as
 * topkv_move_layer(pool view, packed view, ..., window 0). */
topkv_status_t topkv_pack_layer_heads(const topkv_pool_t* src, int32_t layer, int32_t num_reqs,
                                      const int32_t* block_tables, int32_t bt_stride, const int32_t* seq_lens,
                                      int32_t head_begin, int32_t head_count, void* dst, int64_t dst_bytes,
                                      hipStream_t stream);

/* Head-sliced unpack: the inverse, into heads [head_begin, +head_count) of a
 * slot-major pool; the pool's other heads are not written. */
topkv_status_t topkv_unpack_layer_heads(const void* src, int64_t src_bytes, const topkv_pool_t* dst,
                                        int32_t layer, int32_t num_reqs, const int32_t* block_tables,
                                        int32_t bt_stride, const int32_t* seq_lens, int32_t head_begin,
                                        int32_t head_count, hipStream_t stream);

/* Packing for S tensor-parallel receivers in one launch: heads
 * [head_begin, head_begin + head_count) split into S equal runs; shard s (its
 * head_count / S heads, [planes][n_r][head_count / S][dim] per request,
 * requests concatenated) goes to dst + s * shard_bytes.  Same as
 * topkv_move_layer(pool view, packed view with `shards` = S, ..., window 0). */
topkv_status_t topkv_pack_layer_shards(const topkv_pool_t* src, int32_t layer, int32_t num_reqs,
                                      const int32_t* block_tables, int32_t bt_stride, const int32_t* seq_lens,
                                      int32_t head_begin, int32_t head_count, int32_t shards, void* dst,
                                      int64_t shard_bytes, hipStream_t stream);

/* The inverse: S shard buffers (at src + s * shard_bytes) into heads
 * [head_begin, head_begin + head_count) of a slot-major pool. */
topkv_status_t topkv_unpack_layer_shards(const void* src, int64_t shard_bytes, int32_t shards,
                                        const topkv_pool_t* dst, int32_t layer, int32_t num_reqs,
                                        const int32_t* block_tables, int32_t bt_stride, const int32_t* seq_lens,
                                        int32_t head_begin, int32_t head_count, hipStream_t stream);

/* Pool-to-pool re-blocking: every head of layer src_layer of `src` (page size
 * P, tables src_tables) into layer dst_layer of `dst` (page size P', tables
 * dst_tables), with no packed staging buffer.  Both pools have the same
 * planes, heads, head_dim and elem_bytes. */
topkv_status_t topkv_reblock_layer(const topkv_pool_t* src, int32_t src_layer, const int32_t* src_tables,
                                   int32_t src_stride, const topkv_pool_t* dst, int32_t dst_layer,
                                   const int32_t* dst_tables, int32_t dst_stride, int32_t num_reqs,
                                   const int32_t* seq_lens, hipStream_t stream);

/* ---- Fixed-state layers (Section 2.2) ------------------------------------
 * Section 2.2 extends Eq. 1 per layer kind: a linear-attention layer holds,
 * per request, a state whose size does not depend on the sequence length.
 * The state cache keeps one request's state of one layer in a slot:
 *   [num_layers][num_slots][state_bytes] bytes at base (device memory).
 * A packed state batch is the requests' states in request order: request r
 * at bytes [r * state_bytes, (r + 1) * state_bytes).  Bytes are opaque. */
typedef struct topkv_state_pool {
  void*   base;         /* device memory, [num_layers][num_slots][state_bytes] */
  int64_t num_slots;    /* slots per layer, > 0 */
  int64_t state_bytes;  /* one request's state in one layer, > 0 */
  int32_t num_layers;   /* > 0 */
  int32_t reserved;     /* must be 0 */
} topkv_state_pool_t;

/* num_reqs * state_bytes, or -1 for a bad descriptor, num_reqs < 0 or
 * overflow. */
int64_t topkv_packed_state_bytes(const topkv_state_pool_t* pool, int32_t num_reqs);

/* Pack one fixed-state layer of num_reqs requests in one launch.
 *   src:       state cache (host struct describing device memory)
 *   layer:     in [0, src->num_layers)
 *   slots:     device int32[num_reqs], request r's slot; a slot outside
 *              [0, num_slots) is skipped (its bytes of dst are not written)
 *   dst:       device buffer of dst_bytes >= num_reqs * state_bytes bytes
 *   launch:    stream and optional kernel-timestamp events (non-null)
 * num_reqs == 0 launches nothing.  TOPKV_ERR_INVALID_ARG for a bad
 * descriptor, layer, num_reqs < 0, null slots/dst, or dst_bytes too small;
 * TOPKV_ERR_UNSUPPORTED when a state spans 2^31 or more tiles;
 * TOPKV_ERR_LAUNCH if the launch fails.  One kernel on the stream; 16-byte
 * vectors when base, dst and state_bytes are 16-byte multiples, narrower
 * ones otherwise. */
topkv_status_t topkv_pack_state_layer(const topkv_state_pool_t* src, int32_t layer, int32_t num_reqs,
                                      const int32_t* slots, void* dst, int64_t dst_bytes,
                                      const topkv_launch_t* launch);

/* Unpack: request r's state from src into slot slots[r] of layer `layer` of
 * dst; every other slot keeps its contents, and a slot outside the cache is
 * skipped.  Slots must be distinct (two requests naming one slot race).
 * src_bytes >= num_reqs * state_bytes, else TOPKV_ERR_INVALID_ARG; other
 * errors as for topkv_pack_state_layer. */
topkv_status_t topkv_unpack_state_layer(const void* src, int64_t src_bytes, const topkv_state_pool_t* dst,
                                        int32_t layer, int32_t num_reqs, const int32_t* slots,
                                        const topkv_launch_t* launch);

/* Checked path for fixed-state layers: report the slot indices that
 * topkv_pack_state_layer / topkv_unpack_state_layer would skip, and (with
 * check_duplicates != 0) slots named twice in the batch, which an unpack
 * destination must not have (two writers of one slot race).
 *   pool:      geometry only (num_slots); base is not accessed
 *   slots:     device int32[num_reqs]
 *   workspace: device memory of topkv_check_state_workspace_bytes(pool)
 *              bytes (a slot bitmap), cleared by this call; may be null when
 *              check_duplicates == 0
 *   result:    device int32[4], written on the stream: [0] TOPKV_OK or
 *              TOPKV_ERR_BOUNDS, [1] slots out of range, [2] repeated slots,
 *              [3] 0.  Read it after the stream has synchronised.
 * TOPKV_ERR_INVALID_ARG for a bad descriptor, num_reqs < 0, null slots
 * (num_reqs > 0) or result, or a missing or short workspace.  Launches small
 * kernels without synchronising; calls sharing a workspace on overlapping
 * streams race. */
topkv_status_t topkv_check_state_slots(const topkv_state_pool_t* pool, int32_t num_reqs, const int32_t* slots,
                                       int32_t check_duplicates, void* workspace, int64_t workspace_bytes,
                                       int32_t* result, hipStream_t stream);

/* Workspace bytes topkv_check_state_slots needs (num_slots bits in 4-byte
 * words); -1 for a null pool or num_slots <= 0. */
int64_t topkv_check_state_workspace_bytes(const topkv_state_pool_t* pool);

/* Layer shipper (Sec. 5.2: layer l's cache leaves while layers l+1 .. L still
 * compute).  Copies run on the GPU's DMA engines (ROCr asynchronous copies),
 * so they take no compute unit from the kernels still running; a worker
 * thread starts each copy once its `ready` event has completed.  Either
 * direction works: the sender ships packed layers device -> pinned host, the
 * receiver copies them pinned host -> device and unpacks each layer once
 * topkv_dma_wait has returned for its ticket.
 *
 * topkv_dma_create: a shipper for the current HIP device, returned in *out
 *   (owned by the caller; free it with topkv_dma_destroy).  TOPKV_ERR_DEVICE
 *   if the HSA runtime or its signals cannot be set up.
 * topkv_dma_submit: queue a copy of `bytes` from src to dst and return its
 *   ticket (1, 2, 3, ... in submission order) in *ticket.  Both pointers must
 *   lie, with all `bytes`, inside one hipMalloc or hipHostMalloc allocation
 *   (device memory or pinned, mapped host memory), else TOPKV_ERR_BOUNDS; the
 *   ranges must not overlap.  `ready` (may be null) is a recorded event that
 *   marks the moment src holds the data; it must have been recorded before
 *   this call and without hipEventDisableSystemFence, so the producer's writes
 *   are visible to the DMA engine.  bytes == 0 queues an ordering point.
 *   Returns at once; the caller keeps both buffers and the event alive, and
 *   the buffers unchanged, until the ticket completes.
 * topkv_dma_wait: block the calling host thread until every ticket up to and
 *   including `ticket` has completed.  After a failed copy every later wait
 *   and submit returns TOPKV_ERR_DEVICE and queued copies are dropped.
 * topkv_dma_destroy: finish every queued copy, stop the worker, free the
 *   shipper; returns the shipper's status.  No other call on the same shipper
 *   may be in progress or follow it.
 * Any number of host threads may submit and wait on one shipper. */
typedef struct topkv_dma topkv_dma_t;
topkv_status_t topkv_dma_create(topkv_dma_t** out);
topkv_status_t topkv_dma_submit(topkv_dma_t* dma, hipEvent_t ready, void* dst, const void* src,
                                int64_t bytes, int64_t* ticket);
topkv_status_t topkv_dma_wait(topkv_dma_t* dma, int64_t ticket);
topkv_status_t topkv_dma_destroy(topkv_dma_t* dma);

/* Static, human-readable name of a status code (never null). */
const char* topkv_status_string(topkv_status_t status);

#ifdef __cplusplus
}
#endif

#endif /* TOPKV_H_ */
