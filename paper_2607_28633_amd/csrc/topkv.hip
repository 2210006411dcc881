// topkv.hip - HIP kernels (gfx950 / CDNA4) and the C ABI of libtopkv.so:
// per-layer paged KV-cache pack (gather a layer's pages into the contiguous
// [plane][token][head][dim] wire layout) and unpack (scatter it into a pool of
// any page size).  The operation and the layouts are specified in
// include/topkv.h (paper: Sections 3.5, 5.2, 6; Eq. 1 in Section 2.2 and the
// MLA rule of Section 5.3 for sizes).
//
// Design (memory-bound byte movement, no MFMA, no arithmetic on values):
//   * Work item = (request, logical page, plane, tile).  One page of one plane
//     is a single contiguous run of min(P, n - i*P) rows on the pool side and
//     also contiguous on the packed side, so every item is a plain contiguous
//     copy of <= kTile bytes.  Unpack with another page size is the same
//     kernel: its items are the DESTINATION pool's pages, which are again one
//     contiguous run each (the packed form has no pages), so no layout
//     transpose and no LDS staging is needed.
//   * Each lane moves VPT 16-byte vectors: all loads are issued before any
//     store, so a workgroup keeps kTile bytes in flight; the lane->vector
//     mapping (j * kThreads + lane) makes each wave instruction touch one
//     contiguous 1 KiB span (coalesced, full cache lines, no read-for-
//     ownership on the write side).
//   * Batched launches take device-resident seq_lens.  Each workgroup turns
//     them into exclusive prefix sums of tokens and pages with a wave64
//     shuffle scan (results in LDS), then maps its work items to requests by
//     binary search.  The grid is sized from host-known bounds (num_reqs *
//     bt_stride pages) and capped at a few workgroups per CU; workgroups
//     stride over the items.
//   * Device-side table entries and lengths are bounds-checked before any
//     access, so malformed tables cannot make the kernel touch memory outside
//     the pool or packed buffer.
#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>

#include <atomic>
#include <cstdint>

#include "internal.h"
#include "topkv.h"

#ifndef TOPKV_VPT
#define TOPKV_VPT 8           // vectors per lane per tile (16-byte vectors: 32 KiB tiles)
#endif
#ifndef TOPKV_WG_PER_CU
#define TOPKV_WG_PER_CU 8     // persistent grid cap = CUs * this
#endif
#ifndef TOPKV_DIRECT_MAX
#define TOPKV_DIRECT_MAX (1 << 20)  // largest one-shot direct-mapped grid (slots)
#endif
#ifndef TOPKV_WINDOW_PERSISTENT
#define TOPKV_WINDOW_PERSISTENT 1   // windows that keep a small share of the table take the persistent grid
#endif
#ifndef TOPKV_DIRECT_MAX_REQS
#define TOPKV_DIRECT_MAX_REQS 1024  // direct grid: each slot sums the lengths of the requests before its own
#endif
#ifndef TOPKV_NONTEMPORAL
#define TOPKV_NONTEMPORAL 1   // streaming hint on the bulk loads and stores
#endif
#ifndef TOPKV_NT_LOADS
#define TOPKV_NT_LOADS TOPKV_NONTEMPORAL
#endif
#ifndef TOPKV_NT_STORES
#define TOPKV_NT_STORES TOPKV_NONTEMPORAL
#endif
#ifndef TOPKV_ROUTE_SINGLE
#define TOPKV_ROUTE_SINGLE 1  // one whole-request move with a device length runs the layout-move direct grid
#endif
#ifndef TOPKV_XCD_REMAP
#define TOPKV_XCD_REMAP 0     // 1: each XCD takes a contiguous eighth of the direct grid (measured slower)
#endif
#ifndef TOPKV_EARLY_LENS
#define TOPKV_EARLY_LENS 1    // direct grid: earlier requests' lengths load with the slot's own words
#endif
#ifndef TOPKV_DIRECT_LDS_PAD
#define TOPKV_DIRECT_LDS_PAD 0      // dynamic LDS bytes per direct-grid workgroup (caps workgroups per CU)
#endif
#ifndef TOPKV_THREADS
#define TOPKV_THREADS 256     // threads per workgroup (a multiple of 64)
#endif
#ifndef TOPKV_SMALL_THREADS
#define TOPKV_SMALL_THREADS 128  // direct grids over 4-8 KiB page planes (TOPKV_THREADS: off)
#endif
#ifndef TOPKV_ENGINE_GRID_BYTES
#define TOPKV_ENGINE_GRID_BYTES (512ll << 20)  // engine without waits: packed bytes per hardware-dispatched grid
#endif

namespace topkv {

constexpr int kThreads = TOPKV_THREADS;
constexpr int kWaves = kThreads / 64;
constexpr int kSmallThreads = TOPKV_SMALL_THREADS;
static_assert(kSmallThreads % 64 == 0 && kSmallThreads <= kThreads, "small-plane workgroups are whole waves");

template <int B> struct Vec;
template <> struct Vec<16> { typedef unsigned int type __attribute__((ext_vector_type(4))); };
template <> struct Vec<8> { typedef unsigned int type __attribute__((ext_vector_type(2))); };
template <> struct Vec<4> { typedef unsigned int type; };
template <> struct Vec<2> { typedef unsigned short type; };
template <> struct Vec<1> { typedef unsigned char type; };

// Scalar kernel arguments (passed by value in the kernarg segment).  The
// four pointers are separate __restrict__ kernel arguments so the compiler
// can prove the tables are never written and read them through the scalar
// cache.
struct MoveParams {
  int64_t page_bytes;         // planes * page_size * row_bytes
  int64_t plane_bytes;        // page_size * row_bytes
  int64_t packed_cap;         // bytes the packed buffer holds
  int64_t num_pages;          // valid page indices are [0, num_pages)
  int32_t row_bytes;          // heads * head_dim * elem_bytes
  int32_t page_size;          // tokens per page of THIS pool
  int32_t planes;
  int32_t num_reqs;
  int32_t bt_stride;
  int32_t n_single;           // tokens of the single request when seq_lens is null
  int32_t tiles_per_plane;    // ceil(plane_bytes / tile bytes)
  int32_t batched;            // 1: lengths come from device seq_lens
  int32_t window;             // > 0: only the last `window` tokens of each request move
  int32_t z_layers;           // batched direct grid: layers on grid z (z = layer * num_reqs + request)
  int64_t plane_stride;       // single request only: > 0 places plane c at packed + c * plane_stride
  int64_t layer_bytes;        // single request, several layers: pool bytes per layer
  int64_t layer_stride;       // single request, several layers: packed bytes between consecutive layers
};

// First token a windowed layer keeps (window 0 keeps all): the last
// `window` tokens of a request of n tokens.
__device__ __forceinline__ int64_t window_start(int64_t n, int32_t window) {
  return (window > 0 && n > window) ? n - window : 0;
}

__device__ __forceinline__ int32_t uniform(int32_t x) { return __builtin_amdgcn_readfirstlane(x); }

// Two small words that every lane needs, fetched as vector loads issued back
// to back (vector loads retire in order, so one wait covers both), then
// broadcast from lane 0.  Scalar loads of the same words would be waited on
// one at a time, since scalar loads may complete out of order.
__device__ __forceinline__ void load_pair(const int32_t* a, const int32_t* b, int32_t* va, int32_t* vb) {
  const int32_t x = __builtin_nontemporal_load(a);
  const int32_t y = __builtin_nontemporal_load(b);
  *va = uniform(x);
  *vb = uniform(y);
}

// Exclusive prefix sums over requests of kept token counts (lengths clamped,
// then cut to the window) and of the pages those tokens occupy, written to
// LDS: tok[r], pg[r] for r < R with totals at index R, and each request's
// first kept token in st[r].  Tokens ride in the high and pages in the low
// 32 bits of one 64-bit value, so a single wave64 shuffle scan yields both.
__device__ void request_prefix(const MoveParams& p, const int32_t* __restrict__ seq_lens, int32_t* tok,
                               int32_t* pg, int32_t* st, uint64_t* wsum) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t max_tok = (int64_t)p.bt_stride * p.page_size;
  uint64_t carry = 0;
  for (int base = 0; base < p.num_reqs; base += kThreads) {
    const int r = base + threadIdx.x;
    uint64_t v = 0;
    if (r < p.num_reqs) {
      int64_t n = seq_lens[r];
      n = n < 0 ? 0 : (n > max_tok ? max_tok : n);
      const int64_t start = window_start(n, p.window);
      const int64_t cnt = n - start;
      const uint64_t pages = cnt > 0 ? (uint64_t)((n - 1) / p.page_size - start / p.page_size + 1) : 0;
      v = ((uint64_t)cnt << 32) | pages;
      st[r] = (int32_t)start;
    }
    uint64_t x = v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const uint64_t y = __shfl_up(x, d, 64);
      if (lane >= d) x += y;
    }
    if (lane == 63) wsum[wave] = x;
    __syncthreads();
    uint64_t before = carry, chunk = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      if (w < wave) before += wsum[w];
      chunk += wsum[w];
    }
    if (r < p.num_reqs) {
      const uint64_t excl = before + x - v;
      tok[r] = (int32_t)(excl >> 32);
      pg[r] = (int32_t)(excl & 0xffffffffu);
    }
    carry += chunk;
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    tok[p.num_reqs] = (int32_t)(carry >> 32);
    pg[p.num_reqs] = (int32_t)(carry & 0xffffffffu);
  }
  __syncthreads();
}

// A tile is up to NT * VPT vectors of VB bytes, NT the workgroup's threads.
// Lane t handles vectors t, t + NT, ... so each wave instruction covers one
// contiguous span.
template <int VB, int VPT, int NT = kThreads>
__device__ __forceinline__ void load_tile(typename Vec<VB>::type (&v)[VPT], const char* __restrict__ src,
                                          int32_t nv) {
  typedef typename Vec<VB>::type V;
  const V* __restrict__ s = reinterpret_cast<const V*>(src);
  if (nv == NT * VPT) {
#pragma unroll
    for (int j = 0; j < VPT; ++j) {
#if TOPKV_NT_LOADS
      v[j] = __builtin_nontemporal_load(s + j * NT + threadIdx.x);
#else
      v[j] = s[j * NT + threadIdx.x];
#endif
    }
  } else {
    // Ragged tile (1 <= nv < NT * VPT): every lane still issues all VPT
    // loads back to back (indices clamped into the tile, so they stay in
    // bounds); only the stores are predicated.
#pragma unroll
    for (int j = 0; j < VPT; ++j) {
      const int idx = j * NT + threadIdx.x;
      v[j] = s[idx < nv ? idx : nv - 1];
    }
  }
}

template <int VB, int VPT, int NT = kThreads>
__device__ __forceinline__ void store_tile(char* __restrict__ dst, const typename Vec<VB>::type (&v)[VPT],
                                           int32_t nv) {
  typedef typename Vec<VB>::type V;
  V* __restrict__ d = reinterpret_cast<V*>(dst);
  if (nv == NT * VPT) {
#pragma unroll
    for (int j = 0; j < VPT; ++j) {
#if TOPKV_NT_STORES
      __builtin_nontemporal_store(v[j], d + j * NT + threadIdx.x);
#else
      d[j * NT + threadIdx.x] = v[j];
#endif
    }
  } else {
#pragma unroll
    for (int j = 0; j < VPT; ++j) {
      const int idx = j * NT + threadIdx.x;
      if (idx < nv) d[idx] = v[j];
    }
  }
}

template <int VB, int VPT>
__device__ __forceinline__ void copy_tile(char* __restrict__ dst, const char* __restrict__ src, int32_t len) {
  typename Vec<VB>::type v[VPT];
  load_tile<VB, VPT>(v, src, len / VB);
  store_tile<VB, VPT>(dst, v, len / VB);
}

// Sum of the kept token counts of requests [0, r): the token offset of
// request r in the packed batch.  Each wave computes it on its own (lanes
// stride over the lengths, then a butterfly of 32-bit shuffles), so no LDS
// and no barrier are involved.  The host keeps one launch's token capacity
// (num_reqs * bt_stride * page_size) below 2^31, so 32 bits suffice.
// `mine` is seq_lens[lane] for lanes below r, already loaded by the caller.
__device__ __forceinline__ int32_t tokens_before(const int32_t* __restrict__ seq_lens, int32_t r,
                                                 int32_t max_tok, int32_t window, int32_t mine) {
  const int lane = threadIdx.x & 63;
  int32_t s = 0;
  for (int j = lane; j < r; j += 64) {
    int32_t n = j == lane ? mine : seq_lens[j];
    n = n < 0 ? 0 : (n > max_tok ? max_tok : n);
    s += (window > 0 && n > window) ? window : n;
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
  return uniform(s);
}

// Direct mapping: one workgroup per (request, table entry, plane, tile)
// slot, read straight from a 3-D grid (z, y, x) = (r, i, c * tiles + k), so the
// slot's length and page index are independent scalar loads issued at once,
// next to the loads of the earlier lengths that give the request's token
// offset; slots past a request's last page exit.  Used when the slot count is
// small enough for a one-shot grid.
// Workgroup coordinates of the direct grid.  The dispatcher hands linear
// workgroup ids to the 8 XCDs round-robin; with TOPKV_XCD_REMAP the ids are
// permuted so XCD k runs the k-th contiguous eighth of the grid (a bijection
// when the workgroup count is a multiple of 8, else the identity).
__device__ __forceinline__ uint3 grid_block() {
#if TOPKV_XCD_REMAP
  const uint32_t gx = gridDim.x, gy = gridDim.y;
  const uint32_t g = gx * gy * gridDim.z;
  uint32_t l = blockIdx.x + gx * (blockIdx.y + gy * blockIdx.z);
  if ((g & 7u) == 0) l = (l & 7u) * (g >> 3) + (l >> 3);
  const uint32_t xy = l % (gx * gy);
  return make_uint3(xy % gx, xy / gx, l / (gx * gy));
#else
  return make_uint3(blockIdx.x, blockIdx.y, blockIdx.z);
#endif
}

template <int VB, int VPT, bool kPack, bool kBatched, int NT>
__device__ __forceinline__ void move_direct(char* __restrict__ pool, char* __restrict__ packed,
                                            const int32_t* __restrict__ tables,
                                            const int32_t* __restrict__ seq_lens, const MoveParams& p) {
  constexpr int32_t kTile = NT * VPT * VB;
  // grid: z = request (single request: z = layer after the first; a batch
  // over several layers: z = layer * num_reqs + request), y = table entry,
  // x = plane * tiles_per_plane + tile
  const uint3 b = grid_block();
  int32_t r = 0;
  int64_t lz = 0;
  if (!kBatched) {
    lz = (int64_t)b.z;
  } else if (p.z_layers > 1) {
    lz = (int64_t)(b.z / (uint32_t)p.num_reqs);
    r = (int32_t)(b.z - (uint32_t)lz * (uint32_t)p.num_reqs);
  } else {
    r = (int32_t)b.z;
  }
  const int32_t i = b.y;
  const int32_t c = (int32_t)(b.x / (uint32_t)p.tiles_per_plane);
  const int32_t k = (int32_t)(b.x - (uint32_t)c * p.tiles_per_plane);
  const int32_t max_tok = p.bt_stride * p.page_size;   // < 2^31 (host check)

  // This slot's table entry and length, loaded together; with them each lane
  // below r loads one earlier request's length (the request's token offset
  // needs them), so the offset costs no further memory latency.
  int32_t page, n, mine = 0;
  if (kBatched) {
#if TOPKV_EARLY_LENS
    if ((int32_t)(threadIdx.x & 63) < r) mine = __builtin_nontemporal_load(seq_lens + (threadIdx.x & 63));
#endif
    load_pair(tables + (int64_t)r * p.bt_stride + i, seq_lens + r, &page, &n);
#if TOPKV_EARLY_LENS
    asm volatile("" ::"v"(mine));   // keep the load here: not sunk past the exit test below
#else
    if ((int32_t)(threadIdx.x & 63) < r) mine = seq_lens[threadIdx.x & 63];
#endif
  } else {
    page = tables[(int64_t)r * p.bt_stride + i];
    n = p.n_single;
  }
  n = n < 0 ? 0 : (n > max_tok ? max_tok : n);
  const int32_t start = (p.window > 0 && n > p.window) ? n - p.window : 0;   // first kept token
  const int32_t cnt = n - start;
  const int32_t first = i * p.page_size;              // page i holds tokens [first, first + P)
  const int32_t lo = first > start ? first : start;
  const int32_t hi = first + p.page_size < n ? first + p.page_size : n;
  const int64_t run = (int64_t)(hi - lo) * p.row_bytes;
  const int64_t tstart = (int64_t)k * kTile;
  // bitwise, not short-circuit: keeps the table load ahead of the first branch
  const bool live = (hi > lo) & (tstart < run) & (page >= 0) & ((int64_t)page < p.num_pages);
  if (!live) return;
  const int32_t nv = (int32_t)((run - tstart < kTile ? run - tstart : kTile) / VB);
  char* pool_ptr = pool + lz * p.layer_bytes + (int64_t)page * p.page_bytes + (int64_t)c * p.plane_bytes +
                   (int64_t)(lo - first) * p.row_bytes + tstart;
  typename Vec<VB>::type v[VPT];
  // Pack: the pool loads go out before the token offset is known (their
  // addresses do not depend on it), so the offset sum overlaps them.
  if (kPack) load_tile<VB, VPT, NT>(v, pool_ptr, nv);
  const int32_t tok0 = (kBatched && r > 0) ? tokens_before(seq_lens, r, max_tok, p.window, mine) : 0;
  int64_t plane_off, end;
  if (!kBatched && p.plane_stride > 0) {          // caller-placed planes (one request)
    plane_off = (int64_t)c * p.plane_stride;
    end = (int64_t)(p.planes - 1) * p.plane_stride + (int64_t)cnt * p.row_bytes;
  } else {
    plane_off = ((int64_t)tok0 * p.planes + (int64_t)c * cnt) * p.row_bytes;
    end = ((int64_t)tok0 + cnt) * p.planes * p.row_bytes;
  }
  if (end + lz * p.layer_stride > p.packed_cap) return;
  if (kBatched && p.z_layers > 1 && end > p.layer_stride) return;   // stays inside its layer's block
  char* packed_ptr = packed + lz * p.layer_stride + plane_off + (int64_t)(lo - start) * p.row_bytes + tstart;
  if (kPack) {
    store_tile<VB, VPT, NT>(packed_ptr, v, nv);
  } else {
    load_tile<VB, VPT, NT>(v, packed_ptr, nv);
    store_tile<VB, VPT, NT>(pool_ptr, v, nv);
  }
}

// One item of the persistent mapping: page g of the batch's kept pages (in
// request order), plane c, tile k.  tok / pg / st are the LDS prefix sums of
// request_prefix (batched) and are not read for a single request.  The item
// is skipped when its tile lies past the page's run, its request's packed
// block would end past packed_cap, or its table entry is out of range.
template <int VB, int VPT, bool kPack>
__device__ __forceinline__ void strided_item(char* __restrict__ pool, char* __restrict__ packed,
                                             const int32_t* __restrict__ tables, const MoveParams& p,
                                             const int32_t* tok, const int32_t* pg, const int32_t* st,
                                             bool batched, int64_t single_start, int64_t packed_cap, int32_t g,
                                             int32_t c, int32_t k) {
  constexpr int64_t kTile = (int64_t)kThreads * VPT * VB;
  int32_t r = 0, tok0 = 0;
  int64_t start = single_start, cnt = p.n_single - single_start;
  int32_t i = (int32_t)(start / p.page_size) + g;
  if (batched) {
    int lo = 0, hi = p.num_reqs - 1;   // largest r with pg[r] <= g
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (pg[mid] <= g) lo = mid; else hi = mid - 1;
    }
    r = uniform(lo);
    tok0 = uniform(tok[r]);
    cnt = uniform(tok[r + 1] - tok0);
    start = uniform(st[r]);
    i = uniform((int32_t)(start / p.page_size) + g - pg[r]);
  }
  const int64_t n = start + cnt;
  const int64_t first = (int64_t)i * p.page_size;
  const int64_t lo_t = first > start ? first : start;
  const int64_t hi_t = first + p.page_size < n ? first + p.page_size : n;
  const int64_t run = (hi_t - lo_t) * p.row_bytes;
  const int64_t tstart = (int64_t)k * kTile;
  if (tstart >= run) return;
  const bool placed = !batched && p.plane_stride > 0;   // caller-placed planes (one request)
  const int64_t req_end = placed ? (int64_t)(p.planes - 1) * p.plane_stride + cnt * p.row_bytes
                                 : ((int64_t)tok0 + cnt) * p.planes * p.row_bytes;
  if (req_end > packed_cap) return;
  const int32_t page = tables[(int64_t)r * p.bt_stride + i];
  if (page < 0 || (int64_t)page >= p.num_pages) return;
  const int32_t len = (int32_t)(run - tstart < kTile ? run - tstart : kTile);
  char* pool_ptr = pool + (int64_t)page * p.page_bytes + (int64_t)c * p.plane_bytes + (lo_t - first) * p.row_bytes +
                   tstart;
  const int64_t plane_off = placed ? (int64_t)c * p.plane_stride
                                   : ((int64_t)tok0 * p.planes + (int64_t)c * cnt) * p.row_bytes;
  char* packed_ptr = packed + plane_off + (lo_t - start) * p.row_bytes + tstart;
  if (kPack) copy_tile<VB, VPT>(packed_ptr, pool_ptr, len);
  else copy_tile<VB, VPT>(pool_ptr, packed_ptr, len);
}

// Persistent mapping for large batches: every workgroup scans the lengths
// into per-request token and page prefix sums (LDS), then strides over the
// live (request, page, plane, tile) items, locating each item's request by
// binary search.  Work is spread evenly however long the requests are.
// pool: pool base already offset to the layer; packed: packed buffer base;
// tables: [num_reqs][bt_stride]; seq_lens: device [num_reqs] (batched only).
template <int VB, int VPT, bool kPack>
__device__ __forceinline__ void move_strided(char* __restrict__ pool, char* __restrict__ packed,
                                           const int32_t* __restrict__ tables,
                                           const int32_t* __restrict__ seq_lens, const MoveParams& p) {
  extern __shared__ uint64_t lds_u64[];
  uint64_t* wsum = lds_u64;                                      // [kWaves]
  int32_t* tok = reinterpret_cast<int32_t*>(lds_u64 + kWaves);   // [num_reqs + 1]
  int32_t* pg = tok + (p.num_reqs + 1);                          // [num_reqs + 1]
  int32_t* st = pg + (p.num_reqs + 1);                           // [num_reqs + 1]

  const bool batched = p.batched != 0;
  int32_t total_pages;
  const int64_t single_start = window_start(p.n_single, p.window);
  if (batched) {
    request_prefix(p, seq_lens, tok, pg, st, wsum);
    total_pages = pg[p.num_reqs];
  } else {
    total_pages = p.n_single > single_start
                      ? (int32_t)((p.n_single - 1) / p.page_size - single_start / p.page_size + 1) : 0;
  }
  // the host guarantees pages * planes * tiles_per_plane < 2^31
  const uint32_t per_page = (uint32_t)(p.planes * p.tiles_per_plane);
  const uint32_t work = (uint32_t)total_pages * per_page;

  for (uint32_t w = blockIdx.x; w < work; w += gridDim.x) {
    const int32_t g = uniform((int32_t)(w / per_page));
    const int32_t rem = (int32_t)(w - (uint32_t)g * per_page);
    const int32_t c = uniform(rem / p.tiles_per_plane);
    const int32_t k = uniform(rem - c * p.tiles_per_plane);
    strided_item<VB, VPT, kPack>(pool, packed, tables, p, tok, pg, st, batched, single_start, p.packed_cap, g, c,
                                 k);
  }
}

// ---------------------------------------------------------------------------
// Layer engine (Section 5.2: layer l leaves while later layers are still
// being produced, so the unit of transfer is one layer).  One persistent
// launch moves layers [first, first + layers) of a batch: the items of every
// layer in layer order (layer z = w / items-per-layer of the flattened item
// index w), each layer exactly as one batched launch would move it, and a
// layer's items only once its ready word says the layer may move.  The
// per-launch costs of one launch per layer (dispatch, the first table and
// length loads, the drain at the end of each kernel) are paid once per
// range instead of once per layer.
// ---------------------------------------------------------------------------

// How the engine waits.  ready == null: every layer may move at once.
struct EngineWait {
  const uint32_t* ready;     // [layers]: layer z may move once ready[z] has reached epoch
  const uint32_t* cancel;    // optional: non-zero makes waiting waves give up
  int32_t* status;           // non-null when ready is: 0, or why a wave gave up
  int64_t timeout_ticks;     // longest one wait lasts, in wall-clock ticks
  uint32_t epoch;
  int32_t layers;
};

// Wait until layer z may move: layers move in order, so z may move once the
// ready words of every layer up to z have reached the epoch.  *ready_below
// is the first layer not yet seen ready (all before it are); each poll reads
// the 64 words from there (one per lane) and raises *ready_below past the
// run of consecutive ready ones.  The words are read with system-scope
// atomic loads (they may live in host memory or be written by another
// agent), then an acquire fence orders the layer's data loads after the
// word.  Between polls that find nothing new the wave sleeps, longer after
// the first few.  The wait gives up when the cancel word is non-zero
// (TOPKV_ERR_CANCELLED), when it has lasted timeout_ticks
// (TOPKV_ERR_TIMEOUT), or when another wave already gave up (status non-
// zero); the first reason is stored in *status with a compare-and-swap from
// 0, and the caller's wave then exits.  Returns true when layer z may move.
__device__ __forceinline__ bool engine_wait(const EngineWait& e, int32_t z, int32_t* ready_below) {
  const int lane = threadIdx.x & 63;
  const uint64_t t0 = (uint64_t)wall_clock64();
  int32_t below = *ready_below;
  for (int32_t polls = 0;; ++polls) {
    uint32_t word = e.epoch;
    if (below + lane < e.layers)
      word = __hip_atomic_load(const_cast<uint32_t*>(e.ready) + below + lane, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_SYSTEM);
    const uint64_t ok = __ballot((int32_t)(word - e.epoch) >= 0);
    const int32_t run = ~ok ? __builtin_ctzll(~ok) : 64;
    below += run;
    if (below > z) {
      *ready_below = below;
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "");
      return true;
    }
    if (run > 0) continue;        // progress: read the next words at once
    int32_t why = 0;
    if (lane == 0) {
      if (__hip_atomic_load(e.status, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0)
        why = -1;
      else if (e.cancel && __hip_atomic_load(const_cast<uint32_t*>(e.cancel), __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_SYSTEM) != 0)
        why = TOPKV_ERR_CANCELLED;
      else if ((int64_t)((uint64_t)wall_clock64() - t0) > e.timeout_ticks)
        why = TOPKV_ERR_TIMEOUT;
      if (why > 0) atomicCAS(e.status, 0, why);
    }
    if (uniform(why) != 0) return false;
    // short sleeps first (a word that is about to arrive), then long ones
    // (~3 us at 2.4 GHz), so thousands of waiting waves do not keep the
    // fabric busy with polls
    if (polls < 16) __builtin_amdgcn_s_sleep(8);
    else __builtin_amdgcn_s_sleep(127);
  }
}

// One engine item (layer z, page g of the batch's pages, plane c, tile k)
// located from the prefix sums alone: both offsets without the page's own
// term, the table entry to read (-1: nothing to move) and the vectors to
// move (no window: every request keeps all its tokens).
struct EngineItem {
  int64_t pool_off;    // from the first layer's slab, without page * page_bytes
  int64_t packed_off;  // from the packed base
  int32_t tidx;        // r * bt_stride + i, or -1
  int32_t nv;          // vectors of VB bytes
  int32_t z;           // layer of the range
};

template <int VB, int VPT>
__device__ __forceinline__ EngineItem engine_locate(const MoveParams& p, const int32_t* tok, const int32_t* pg,
                                                    uint32_t w, uint32_t work, uint32_t per_page, int32_t layers) {
  constexpr int64_t kTile = (int64_t)kThreads * VPT * VB;
  EngineItem it;
  const int32_t z = uniform((int32_t)(w / work));
  const uint32_t item = w - (uint32_t)z * work;
  const int32_t g = uniform((int32_t)(item / per_page));
  const int32_t rem = (int32_t)(item - (uint32_t)g * per_page);
  const int32_t c = uniform(rem / p.tiles_per_plane);
  const int32_t k = uniform(rem - c * p.tiles_per_plane);
  int lo = 0, hi = p.num_reqs - 1;   // largest r with pg[r] <= g
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (pg[mid] <= g) lo = mid; else hi = mid - 1;
  }
  const int32_t r = uniform(lo);
  const int32_t tok0 = uniform(tok[r]);
  const int32_t n = uniform(tok[r + 1] - tok0);
  const int32_t i = uniform(g - pg[r]);
  const int64_t first = (int64_t)i * p.page_size;
  const int64_t last = first + p.page_size < n ? first + p.page_size : n;
  const int64_t run = (last - first) * p.row_bytes;
  const int64_t tstart = (int64_t)k * kTile;
  const int64_t off = (int64_t)z * p.layer_stride;
  int64_t cap = p.packed_cap - off;
  if (layers > 1 && cap > p.layer_stride) cap = p.layer_stride;
  const int64_t req_end = ((int64_t)tok0 + n) * p.planes * p.row_bytes;
  it.z = z;
  it.tidx = (tstart < run && req_end <= cap) ? r * p.bt_stride + i : -1;
  it.nv = (int32_t)((run - tstart < kTile ? run - tstart : kTile) / VB);
  it.pool_off = (int64_t)z * p.layer_bytes + (int64_t)c * p.plane_bytes + tstart;
  it.packed_off = off + (((int64_t)tok0 * p.planes + (int64_t)c * n) + first) * p.row_bytes + tstart;
  return it;
}

// The item's source and destination once its table entry is known; returns
// the vectors to move (0: skipped, entry outside the pool or -1).
template <bool kPack>
__device__ __forceinline__ int32_t engine_address(const EngineItem& it, int32_t page, const MoveParams& p,
                                                  char* pool, char* packed, const char** src, char** dst) {
  if (it.tidx < 0 || page < 0 || (int64_t)page >= p.num_pages) return 0;
  char* pool_ptr = pool + (int64_t)page * p.page_bytes + it.pool_off;
  char* packed_ptr = packed + it.packed_off;
  *src = kPack ? pool_ptr : packed_ptr;
  *dst = kPack ? packed_ptr : pool_ptr;
  return it.nv;
}

// pool: the first layer's slab; packed: layer z's block starts at packed +
// z * layer_stride and holds min(layer_stride, packed_cap - z * layer_stride)
// bytes (packed_cap alone for one layer).  Workgroup b runs items b,
// b + gridDim.x, ... so the whole grid works through the layers in order
// (a few layers in flight at a time).
template <int VB, int VPT, bool kPack>
__global__ __launch_bounds__(kThreads) void kv_engine_kernel(char* __restrict__ pool, char* __restrict__ packed,
                                                             const int32_t* __restrict__ tables,
                                                             const int32_t* __restrict__ seq_lens, MoveParams p,
                                                             EngineWait e) {
  extern __shared__ uint64_t lds_u64[];
  uint64_t* wsum = lds_u64;
  int32_t* tok = reinterpret_cast<int32_t*>(lds_u64 + kWaves);
  int32_t* pg = tok + (p.num_reqs + 1);
  int32_t* st = pg + (p.num_reqs + 1);
  request_prefix(p, seq_lens, tok, pg, st, wsum);
  const uint32_t per_page = (uint32_t)(p.planes * p.tiles_per_plane);
  const uint32_t work = (uint32_t)pg[p.num_reqs] * per_page;     // items per layer
  // the host keeps layers * num_reqs * bt_stride * per_page below 2^31
  const uint32_t total = work * (uint32_t)e.layers;
  int32_t ready_below = e.ready ? 0 : e.layers;
  for (uint32_t w = blockIdx.x; w < total; w += gridDim.x) {
    const EngineItem it = engine_locate<VB, VPT>(p, tok, pg, w, work, per_page, e.layers);
    if (it.z >= ready_below && !engine_wait(e, it.z, &ready_below)) return;
    const char* src = nullptr;
    char* dst = nullptr;
    const int32_t nv = engine_address<kPack>(it, it.tidx >= 0 ? tables[it.tidx] : -1, p, pool, packed, &src, &dst);
    if (nv) copy_tile<VB, VPT>(dst, src, nv * VB);
  }
}

// kMode: 0 = persistent (strided) grid, 1 = direct grid for one request with
// a host-side length, 2 = direct grid for a batch with device lengths.
enum { kStrided = 0, kDirectSingle = 1, kDirectBatched = 2 };

// VB: bytes per vector (16 on the fast path); VPT: vectors per lane per tile;
// NT: threads per workgroup (kThreads, or kSmallThreads for direct grids over
// small page planes), so a tile is NT * VPT * VB bytes (chosen per launch to
// fit a page plane).  The persistent grid runs kThreads only.
template <int VB, int VPT, int kMode, int NT>
__global__ __launch_bounds__(NT) void kv_pack_kernel(char* __restrict__ pool, char* __restrict__ packed,
                                                     const int32_t* __restrict__ tables,
                                                     const int32_t* __restrict__ seq_lens, MoveParams p) {
  static_assert(kMode != kStrided || NT == kThreads, "the persistent grid runs kThreads-wide workgroups");
  if (kMode == kStrided) move_strided<VB, VPT, true>(pool, packed, tables, seq_lens, p);
  else move_direct<VB, VPT, true, kMode == kDirectBatched, NT>(pool, packed, tables, seq_lens, p);
}

template <int VB, int VPT, int kMode, int NT>
__global__ __launch_bounds__(NT) void kv_unpack_kernel(char* __restrict__ pool, char* __restrict__ packed,
                                                       const int32_t* __restrict__ tables,
                                                       const int32_t* __restrict__ seq_lens, MoveParams p) {
  static_assert(kMode != kStrided || NT == kThreads, "the persistent grid runs kThreads-wide workgroups");
  if (kMode == kStrided) move_strided<VB, VPT, false>(pool, packed, tables, seq_lens, p);
  else move_direct<VB, VPT, false, kMode == kDirectBatched, NT>(pool, packed, tables, seq_lens, p);
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------

constexpr int kMaxDevices = 64;
std::atomic<int> g_cu_count[kMaxDevices];

topkv_status_t cu_count(int* out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return TOPKV_ERR_DEVICE;
  if (dev < kMaxDevices) {
    const int cached = g_cu_count[dev].load(std::memory_order_relaxed);
    if (cached > 0) { *out = cached; return TOPKV_OK; }
  }
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    return TOPKV_ERR_DEVICE;
  if (dev < kMaxDevices) g_cu_count[dev].store(cus, std::memory_order_relaxed);
  *out = cus;
  return TOPKV_OK;
}

struct Geometry {
  int64_t row_bytes, plane_bytes, page_bytes, layer_bytes;
};

topkv_status_t pool_geometry(const topkv_pool_t* pool, int32_t layer, Geometry* g) {
  if (!pool || !pool->base) return TOPKV_ERR_INVALID_ARG;
  if (pool->num_pages <= 0 || pool->num_layers <= 0 || pool->page_size <= 0 || pool->planes <= 0 ||
      pool->num_heads <= 0 || pool->head_dim <= 0)
    return TOPKV_ERR_INVALID_ARG;
  if (pool->elem_bytes != 1 && pool->elem_bytes != 2 && pool->elem_bytes != 4 && pool->elem_bytes != 8)
    return TOPKV_ERR_INVALID_ARG;
  if (layer < 0 || layer >= pool->num_layers) return TOPKV_ERR_INVALID_ARG;
  int64_t row, plane, page, lay, all;
  if (__builtin_mul_overflow((int64_t)pool->num_heads, (int64_t)pool->head_dim, &row) ||
      __builtin_mul_overflow(row, (int64_t)pool->elem_bytes, &row) ||
      __builtin_mul_overflow(row, (int64_t)pool->page_size, &plane) ||
      __builtin_mul_overflow(plane, (int64_t)pool->planes, &page) ||
      __builtin_mul_overflow(page, pool->num_pages, &lay) ||
      __builtin_mul_overflow(lay, (int64_t)pool->num_layers, &all))
    return TOPKV_ERR_UNSUPPORTED;
  if (row > INT32_MAX || pool->num_pages > INT32_MAX) return TOPKV_ERR_UNSUPPORTED;
  g->row_bytes = row;
  g->plane_bytes = plane;
  g->page_bytes = page;
  g->layer_bytes = lay;
  return TOPKV_OK;
}

int vector_bytes(uintptr_t a, uintptr_t b, int64_t row) {
  for (int vb = 16; vb > 1; vb >>= 1)
    if (a % vb == 0 && b % vb == 0 && row % vb == 0) return vb;
  return 1;
}

typedef void (*KernelFn)(char*, char*, const int32_t*, const int32_t*, MoveParams);

template <int VB, int VPT, int kMode, int NT = kThreads>
KernelFn kernel_for(bool pack) {
  return pack ? kv_pack_kernel<VB, VPT, kMode, NT> : kv_unpack_kernel<VB, VPT, kMode, NT>;
}

template <int kMode>
KernelFn pick_kernel_mode(bool pack, int vb, int vpt) {
  switch (vb) {
    case 16:
      if (vpt == TOPKV_VPT) return kernel_for<16, TOPKV_VPT, kMode>(pack);
      switch (vpt) {
        case 8: return kernel_for<16, 8, kMode>(pack);
        case 4: return kernel_for<16, 4, kMode>(pack);
        case 2: return kernel_for<16, 2, kMode>(pack);
        default: return kernel_for<16, 1, kMode>(pack);
      }
    case 8: return kernel_for<8, TOPKV_VPT, kMode>(pack);
    case 4: return kernel_for<4, TOPKV_VPT, kMode>(pack);
    case 2: return kernel_for<2, TOPKV_VPT, kMode>(pack);
    default: return kernel_for<1, TOPKV_VPT, kMode>(pack);
  }
}

// threads: kThreads, or kSmallThreads as launch_threads chose it (then the
// tile is 2 vectors of 16 bytes per lane; null for any other combination).
KernelFn pick_kernel(bool pack, int vb, int vpt, bool direct, bool batched, int threads = kThreads) {
  if (threads != kThreads) {
    if (!direct || vb != 16 || vpt != 2 || threads != kSmallThreads) return nullptr;
    return batched ? kernel_for<16, 2, kDirectBatched, kSmallThreads>(pack)
                   : kernel_for<16, 2, kDirectSingle, kSmallThreads>(pack);
  }
  if (!direct) return pick_kernel_mode<kStrided>(pack, vb, vpt);
  return batched ? pick_kernel_mode<kDirectBatched>(pack, vb, vpt) : pick_kernel_mode<kDirectSingle>(pack, vb, vpt);
}

// Vectors per lane for 16-byte vectors: the largest of TOPKV_VPT, 4, 2, 1
// whose tile of `threads` lanes still fits in one page plane, so small planes
// (e.g. 16 KiB for 1 KiB rows in 16-token pages) get full tiles instead of
// half-empty ones.
int vectors_per_lane(int vb, int64_t plane_bytes, int threads = kThreads) {
  if (vb != 16) return TOPKV_VPT;
  for (int v = TOPKV_VPT; v > 1; v >>= 1)
    if ((int64_t)threads * v * 16 <= plane_bytes) return v;
  return 1;
}

// Threads per workgroup of a launch.  A direct grid over page planes of 4 to
// 8 KiB (one KV head of 128 bf16 in 16-token pages: 4 KiB) runs
// kSmallThreads-wide workgroups with two 16-byte vectors per lane, where
// kThreads lanes would hold one vector each: half the waves per tile, each
// with twice the loads in flight.  Pack and unpack both take it (a pack
// grid runs at its best after an unpack grid of the same width).  Larger
// planes, and the persistent grid, run kThreads.
int launch_threads(bool direct, int vb, int64_t plane_bytes) {
  if (direct && vb == 16 && kSmallThreads < kThreads && plane_bytes >= (int64_t)kSmallThreads * 2 * 16 &&
      plane_bytes < (int64_t)kThreads * 2 * 16)
    return kSmallThreads;
  return kThreads;
}

// launch_threads for a launch whose grid is already laid out in tiles of
// `tile` bytes (kThreads lanes): the narrower workgroup is taken only when its
// own tile has the same size, so the grid and tiles_per_plane stand.
int narrow_threads(bool direct, int vb, int64_t plane_bytes, int64_t tile) {
  const int t = launch_threads(direct, vb, plane_bytes);
  return (int64_t)t * vectors_per_lane(vb, plane_bytes, t) * vb == tile ? t : kThreads;
}

// Shared launcher for the four movement entry points.
//   pack:     direction (pool -> packed when true)
//   seq_lens: device lengths (batched) or null (single request of n_single)
topkv_status_t launch_move(bool pack, const topkv_pool_t* pool, int32_t layer, void* packed,
                           int64_t packed_cap, int32_t num_reqs, const int32_t* tables,
                           int32_t bt_stride, const int32_t* seq_lens, int32_t n_single, int32_t window,
                           int64_t plane_stride, const topkv_launch_t* launch, int32_t layers = 1,
                           int64_t layer_stride = 0) {
  Geometry g;
  topkv_status_t st = pool_geometry(pool, layer, &g);
  if (st != TOPKV_OK) return st;
  if (!launch) return TOPKV_ERR_INVALID_ARG;
  if (num_reqs < 0 || n_single < 0 || packed_cap < 0 || window < 0 || plane_stride < 0) return TOPKV_ERR_INVALID_ARG;
  if (plane_stride > 0 && seq_lens) return TOPKV_ERR_INVALID_ARG;   // placed planes: one request only
  // several layers in one launch: one request with placed planes, layers [layer, layer + layers)
  if (layers < 1 || layer_stride < 0 || (int64_t)layer + layers > pool->num_layers) return TOPKV_ERR_INVALID_ARG;
  if (layers > 1 && (seq_lens || plane_stride <= 0 || layers > 65535)) return TOPKV_ERR_INVALID_ARG;
  if (num_reqs > TOPKV_MAX_BATCH_REQS) return TOPKV_ERR_UNSUPPORTED;
  if (num_reqs == 0 || (!seq_lens && n_single == 0)) return TOPKV_OK;  // nothing to move
  if (!tables || !packed || bt_stride <= 0) return TOPKV_ERR_INVALID_ARG;
  // a host-side length must fit its table
  if (!seq_lens && ((int64_t)n_single + pool->page_size - 1) / pool->page_size > bt_stride)
    return TOPKV_ERR_INVALID_ARG;

  if (topkv_internal::checked_mode()) {
    // packed bytes per kept token, and (placed planes) the bytes before the last plane's rows
    const int64_t per_token = plane_stride > 0 ? g.row_bytes : (int64_t)pool->planes * g.row_bytes;
    int64_t fixed = 0, planes_before = 0;
    if (plane_stride > 0 && (__builtin_mul_overflow((int64_t)(layers - 1), layer_stride, &fixed) ||
                             __builtin_mul_overflow((int64_t)(pool->planes - 1), plane_stride, &planes_before) ||
                             __builtin_add_overflow(fixed, planes_before, &fixed)))
      return TOPKV_ERR_UNSUPPORTED;
    st = topkv_internal::checked_tables(pool, seq_lens ? num_reqs : 1, tables, bt_stride, seq_lens, n_single,
                                        window, !pack, per_token, fixed, packed_cap, launch->stream);
    if (st != TOPKV_OK) return st;
  }

  // One request, every token kept, planes in the packed order: the
  // layout-move kernel's one-request grid does the same copy with less index
  // work per piece.  A device length needs a packed buffer large enough for
  // the whole table (that grid skips pieces past the buffer's end, where this
  // kernel leaves an overrunning request unmoved); a host length is checked
  // against the buffer here.
  const int64_t route_tok = seq_lens ? (int64_t)bt_stride * pool->page_size : n_single;
  int64_t route_rows, route_bytes;
  const bool fits = !__builtin_mul_overflow((int64_t)pool->planes, route_tok, &route_rows) &&
                    !__builtin_mul_overflow(route_rows, g.row_bytes, &route_bytes) && route_bytes <= packed_cap &&
                    route_tok <= (int64_t)bt_stride * pool->page_size;
  if (TOPKV_ROUTE_SINGLE && num_reqs == 1 && window == 0 && plane_stride == 0 && layers == 1 && fits) {
    bool launched = false;
    st = topkv_internal::single_request_move(pack, pool, layer, packed, packed_cap, tables, bt_stride, seq_lens,
                                             n_single, launch, &launched);
    if (st != TOPKV_OK || launched) return st;
  }

  int vb = vector_bytes(reinterpret_cast<uintptr_t>(pool->base), reinterpret_cast<uintptr_t>(packed), g.row_bytes);
  while (plane_stride % vb || layer_stride % vb) vb >>= 1;   // placed planes keep every run vector-aligned
  const int vpt = vectors_per_lane(vb, g.plane_bytes);
  const int64_t tile = (int64_t)kThreads * vpt * vb;
  const int64_t tpp = (g.plane_bytes + tile - 1) / tile;
  int64_t per_page, max_pages, work;
  if (seq_lens) {
    max_pages = (int64_t)num_reqs * bt_stride;
  } else {
    max_pages = ((int64_t)n_single + pool->page_size - 1) / pool->page_size;   // <= bt_stride (checked above)
  }
  // one launch's token capacity (requests x table width x page size) must stay below 2^31
  const int64_t tok_cap = (seq_lens ? (int64_t)num_reqs : 1) * bt_stride * (int64_t)pool->page_size;
  if (__builtin_mul_overflow(tpp, (int64_t)pool->planes, &per_page) || per_page > INT32_MAX ||
      __builtin_mul_overflow(max_pages, per_page, &work) || work > INT32_MAX || tok_cap > INT32_MAX)
    return TOPKV_ERR_UNSUPPORTED;

  // Direct mapping when every (request, table entry, plane, tile) slot can
  // get its own workgroup; otherwise a persistent grid over the live items.
  const int64_t reqs = seq_lens ? (int64_t)num_reqs : 1;
  const int64_t slots = reqs * bt_stride * per_page;
  // A window keeps at most ceil(window / P) + 1 pages of each request; when that is a small share of
  // the table, a direct grid would be mostly slots that exit at once, so the persistent grid (which
  // visits live items only) takes the launch.
  const int64_t win_pages = window > 0 ? ((int64_t)window + pool->page_size - 1) / pool->page_size + 1 : bt_stride;
  const bool sparse = TOPKV_WINDOW_PERSISTENT && seq_lens && win_pages * 4 <= bt_stride;
  const bool direct = !sparse && slots <= TOPKV_DIRECT_MAX && bt_stride <= 65535 && reqs <= TOPKV_DIRECT_MAX_REQS;
  dim3 grid3;
  unsigned grid = 0;
  if (layers > 1 && !direct) return TOPKV_ERR_UNSUPPORTED;   // the caller moves one layer per launch instead
  if (direct) {
    grid3 = dim3((unsigned)per_page, (unsigned)bt_stride, (unsigned)(seq_lens ? reqs : layers));
    grid = (unsigned)slots;
  } else {
    int cus = 0;
    st = cu_count(&cus);
    if (st != TOPKV_OK) return st;
    const int64_t cap = (int64_t)cus * TOPKV_WG_PER_CU;
    grid = (unsigned)(work < cap ? work : cap);
    grid3 = dim3(grid);
  }
  if (grid == 0) return TOPKV_OK;

  char* pool_ptr = static_cast<char*>(pool->base) + (int64_t)layer * g.layer_bytes;
  char* packed_ptr = static_cast<char*>(packed);
  MoveParams p;
  p.page_bytes = g.page_bytes;
  p.plane_bytes = g.plane_bytes;
  p.packed_cap = packed_cap;
  p.num_pages = pool->num_pages;
  p.row_bytes = (int32_t)g.row_bytes;
  p.page_size = pool->page_size;
  p.planes = pool->planes;
  p.num_reqs = seq_lens ? num_reqs : 1;
  p.bt_stride = bt_stride;
  p.n_single = n_single;
  p.tiles_per_plane = (int32_t)tpp;
  p.batched = seq_lens ? 1 : 0;
  p.window = window;
  p.z_layers = 1;
  p.plane_stride = plane_stride;
  p.layer_bytes = g.layer_bytes;
  p.layer_stride = layer_stride;

  const size_t lds = (seq_lens && !direct) ? sizeof(uint64_t) * kWaves + sizeof(int32_t) * 3 * ((size_t)num_reqs + 1)
                                           : (direct ? (size_t)TOPKV_DIRECT_LDS_PAD : 0);
  void* args[] = {&pool_ptr, &packed_ptr, &tables, &seq_lens, &p};
  const int threads = narrow_threads(direct, vb, g.plane_bytes, tile);
  const void* fn = reinterpret_cast<const void*>(
      pick_kernel(pack, vb, vectors_per_lane(vb, g.plane_bytes, threads), direct, seq_lens != nullptr, threads));
  if (!fn) return TOPKV_ERR_UNSUPPORTED;
  hipError_t e;
  if (launch->start || launch->stop)
    e = hipExtLaunchKernel(fn, grid3, dim3(threads), args, lds, launch->stream, launch->start,
                           launch->stop, 0);
  else
    e = hipLaunchKernel(fn, grid3, dim3(threads), args, lds, launch->stream);
  return e == hipSuccess ? TOPKV_OK : TOPKV_ERR_LAUNCH;
}

#ifndef TOPKV_ENGINE_WG_PER_CU
#define TOPKV_ENGINE_WG_PER_CU 8   // layer engine: default workgroups kept per compute unit
#endif

typedef void (*EngineFn)(char*, char*, const int32_t*, const int32_t*, MoveParams, EngineWait);

template <int VB, int VPT>
EngineFn engine_for(bool pack) {
  return pack ? kv_engine_kernel<VB, VPT, true> : kv_engine_kernel<VB, VPT, false>;
}

EngineFn pick_engine(bool pack, int vb, int vpt) {
  switch (vb) {
    case 16:
      switch (vpt) {
        case 8: return engine_for<16, 8>(pack);
        case 4: return engine_for<16, 4>(pack);
        case 2: return engine_for<16, 2>(pack);
        default: return engine_for<16, 1>(pack);
      }
    case 8: return engine_for<8, TOPKV_VPT>(pack);
    case 4: return engine_for<4, TOPKV_VPT>(pack);
    case 2: return engine_for<2, TOPKV_VPT>(pack);
    default: return engine_for<1, TOPKV_VPT>(pack);
  }
}

// Wall-clock ticks per microsecond of the current device (the clock the
// kernels read with wall_clock64), cached per device.
std::atomic<int> g_clock_khz[kMaxDevices];

topkv_status_t wall_clock_khz(int* out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return TOPKV_ERR_DEVICE;
  if (dev < kMaxDevices) {
    const int cached = g_clock_khz[dev].load(std::memory_order_relaxed);
    if (cached > 0) { *out = cached; return TOPKV_OK; }
  }
  int khz = 0;
  if (hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess || khz <= 0)
    return TOPKV_ERR_DEVICE;
  if (dev < kMaxDevices) g_clock_khz[dev].store(khz, std::memory_order_relaxed);
  *out = khz;
  return TOPKV_OK;
}

// Layers per hardware-dispatched grid of an engine call that does not wait:
// the caller's count when it sets one, else the range cut into
// ceil(layers * layer_stride / TOPKV_ENGINE_GRID_BYTES) grids of equal layer
// count (the last one fewer).  One grid over a long range ran slower than
// several shorter grids back to back on MI355X: 80 layers of 16 MiB packed
// 1.2% slower than 3 grids of 27, 80 layers of 140 MB 2.7% (scattered pages)
// to 7.8% (contiguous pages) slower than grids of 3 to 4, with the step
// fastest from about 256 MiB to 1 GiB of packed blocks per grid.
int32_t engine_layers_per_grid(int32_t layers, int64_t layer_stride, const topkv_engine_t* opt) {
  if (opt && opt->layers_per_grid > 0) return opt->layers_per_grid < layers ? opt->layers_per_grid : layers;
  if (layers <= 1 || layer_stride <= 0) return layers;
  int64_t bytes;
  if (__builtin_mul_overflow((int64_t)layers, layer_stride, &bytes)) return 1;
  const int64_t grids = bytes / TOPKV_ENGINE_GRID_BYTES + (bytes % TOPKV_ENGINE_GRID_BYTES != 0);
  return (int32_t)(((int64_t)layers + grids - 1) / grids);
}

// The layer engine's launcher (both directions).  The argument rules are
// those of the batched calls applied to every layer of the range, plus the
// range, the layer stride and the wait options.
topkv_status_t engine_move(bool pack, const topkv_pool_t* pool, int32_t first_layer, int32_t layers,
                           void* packed, int64_t packed_cap, int64_t layer_stride, int32_t num_reqs,
                           const int32_t* tables, int32_t bt_stride, const int32_t* seq_lens,
                           const topkv_engine_t* opt, hipStream_t stream) {
  Geometry g;
  topkv_status_t st = pool_geometry(pool, first_layer, &g);
  if (st != TOPKV_OK) return st;
  if (layers < 1 || (int64_t)first_layer + layers > pool->num_layers) return TOPKV_ERR_INVALID_ARG;
  if (num_reqs < 0 || packed_cap < 0 || layer_stride < 0 || (layers > 1 && layer_stride == 0))
    return TOPKV_ERR_INVALID_ARG;
  int64_t before_last;
  if (__builtin_mul_overflow((int64_t)(layers - 1), layer_stride, &before_last) || before_last > packed_cap)
    return TOPKV_ERR_INVALID_ARG;
  const bool waits = opt && opt->ready;
  if (waits && (!opt->status || opt->timeout_us <= 0 || opt->timeout_us > 60000000)) return TOPKV_ERR_INVALID_ARG;
  if (opt && (opt->workgroups_per_cu < 0 || opt->workgroups_per_cu > 64 || opt->layers_per_grid < 0))
    return TOPKV_ERR_INVALID_ARG;
  if (num_reqs > TOPKV_MAX_BATCH_REQS) return TOPKV_ERR_UNSUPPORTED;
  if (num_reqs == 0) return TOPKV_OK;
  if (!tables || !seq_lens || !packed || bt_stride <= 0) return TOPKV_ERR_INVALID_ARG;

  if (topkv_internal::checked_mode()) {
    // the last layer's block is the smallest
    int64_t cap = packed_cap - before_last;
    if (layers > 1 && cap > layer_stride) cap = layer_stride;
    st = topkv_internal::checked_tables(pool, num_reqs, tables, bt_stride, seq_lens, 0, 0, !pack,
                                        (int64_t)pool->planes * g.row_bytes, 0, cap, stream);
    if (st != TOPKV_OK) return st;
  }

  int vb = vector_bytes(reinterpret_cast<uintptr_t>(pool->base), reinterpret_cast<uintptr_t>(packed), g.row_bytes);
  while (layer_stride % vb) vb >>= 1;
  const int vpt = vectors_per_lane(vb, g.plane_bytes);
  const int64_t tile = (int64_t)kThreads * vpt * vb;
  const int64_t tpp = (g.plane_bytes + tile - 1) / tile;
  int64_t per_page, work, total;
  const int64_t tok_cap = (int64_t)num_reqs * bt_stride * (int64_t)pool->page_size;
  if (__builtin_mul_overflow(tpp, (int64_t)pool->planes, &per_page) || per_page > INT32_MAX ||
      __builtin_mul_overflow((int64_t)num_reqs * bt_stride, per_page, &work) ||
      __builtin_mul_overflow(work, (int64_t)layers, &total) || total > INT32_MAX || tok_cap > INT32_MAX)
    return TOPKV_ERR_UNSUPPORTED;

  char* pool_ptr = static_cast<char*>(pool->base) + (int64_t)first_layer * g.layer_bytes;
  char* packed_ptr = static_cast<char*>(packed);
  MoveParams p;
  p.page_bytes = g.page_bytes;
  p.plane_bytes = g.plane_bytes;
  p.packed_cap = packed_cap;
  p.num_pages = pool->num_pages;
  p.row_bytes = (int32_t)g.row_bytes;
  p.page_size = pool->page_size;
  p.planes = pool->planes;
  p.num_reqs = num_reqs;
  p.bt_stride = bt_stride;
  p.n_single = 0;
  p.tiles_per_plane = (int32_t)tpp;
  p.batched = 1;
  p.window = 0;
  p.z_layers = 1;
  p.plane_stride = 0;
  p.layer_bytes = g.layer_bytes;
  p.layer_stride = layer_stride;

  // Every layer ready at launch: the batched direct grid with the layers on
  // grid z (z = layer * num_reqs + request), dispatched by the hardware - no
  // waiting, so nothing needs to stay resident.  Same slot rules as one
  // batched launch (slots past a request's pages exit at once).  The range
  // goes out as consecutive grids of engine_layers_per_grid layers each:
  // grid j starts at layer j * per with its pool and packed pointers moved
  // there, and its capacity is what the whole range allows those layers
  // (packed_cap less the layers before it; with several layers in the call
  // at most per * layer_stride, so a one-layer grid keeps each layer's
  // block within layer_stride as a longer grid does).
  if (!waits && work <= TOPKV_DIRECT_MAX && bt_stride <= 65535 && num_reqs <= TOPKV_DIRECT_MAX_REQS &&
      (int64_t)num_reqs * layers <= 65535) {
    const int32_t per = engine_layers_per_grid(layers, layer_stride, opt);
    const int threads = narrow_threads(true, vb, g.plane_bytes, tile);
    const void* fn = reinterpret_cast<const void*>(
        pick_kernel(pack, vb, vectors_per_lane(vb, g.plane_bytes, threads), true, true, threads));
    if (!fn) return TOPKV_ERR_UNSUPPORTED;
    for (int32_t j = 0; j < layers; j += per) {
      const int32_t n = layers - j < per ? layers - j : per;
      MoveParams q = p;
      q.z_layers = n;
      q.packed_cap = packed_cap - (int64_t)j * layer_stride;          // >= 0: j <= layers - 1
      int64_t span;   // this grid's layers' blocks, n * layer_stride
      if (layers > 1 && !__builtin_mul_overflow((int64_t)n, layer_stride, &span) && q.packed_cap > span)
        q.packed_cap = span;
      char* pool_j = pool_ptr + (int64_t)j * g.layer_bytes;
      char* packed_j = packed_ptr + (int64_t)j * layer_stride;
      void* args[] = {&pool_j, &packed_j, &tables, &seq_lens, &q};
      const dim3 grid3((unsigned)per_page, (unsigned)bt_stride, (unsigned)(num_reqs * n));
      if (hipLaunchKernel(fn, grid3, dim3(threads), args, (size_t)TOPKV_DIRECT_LDS_PAD, stream) != hipSuccess)
        return TOPKV_ERR_LAUNCH;
    }
    return TOPKV_OK;
  }

  int cus = 0;
  st = cu_count(&cus);
  if (st != TOPKV_OK) return st;
  const int per_cu = (opt && opt->workgroups_per_cu > 0) ? opt->workgroups_per_cu : TOPKV_ENGINE_WG_PER_CU;
  const int64_t cap_grid = (int64_t)cus * per_cu;
  const unsigned grid = (unsigned)(total < cap_grid ? total : cap_grid);
  if (grid == 0) return TOPKV_OK;

  EngineWait e;
  e.ready = waits ? opt->ready : nullptr;
  e.cancel = waits ? opt->cancel : nullptr;
  e.status = waits ? opt->status : nullptr;
  e.epoch = waits ? opt->epoch : 0;
  e.layers = layers;
  e.timeout_ticks = 0;
  if (waits) {
    int khz = 0;
    st = wall_clock_khz(&khz);
    if (st != TOPKV_OK) return st;
    e.timeout_ticks = opt->timeout_us * (int64_t)khz / 1000;
  }

  const size_t lds = sizeof(uint64_t) * kWaves + sizeof(int32_t) * 3 * ((size_t)num_reqs + 1);
  void* args[] = {&pool_ptr, &packed_ptr, &tables, &seq_lens, &p, &e};
  const void* fn = reinterpret_cast<const void*>(pick_engine(pack, vb, vpt));
  return hipLaunchKernel(fn, dim3(grid), dim3(kThreads), args, lds, stream) == hipSuccess ? TOPKV_OK
                                                                                         : TOPKV_ERR_LAUNCH;
}

int64_t single_bytes(const topkv_pool_t* pool, int32_t n) {
  int64_t b;
  if (__builtin_mul_overflow((int64_t)pool->num_heads, (int64_t)pool->head_dim, &b) ||
      __builtin_mul_overflow(b, (int64_t)pool->elem_bytes, &b) ||
      __builtin_mul_overflow(b, (int64_t)pool->planes * n, &b))
    return -1;
  return b;
}

}  // namespace topkv

namespace topkv_internal {

topkv_status_t pool_ok(const topkv_pool_t* pool) {
  topkv::Geometry g;
  return topkv::pool_geometry(pool, 0, &g);
}

topkv_status_t placed_layers_move(bool pack, const topkv_pool_t* pool, int32_t first_layer, int32_t layers,
                                  void* packed, int64_t packed_cap, int64_t plane_stride, int64_t layer_stride,
                                  const int32_t* block_table, int32_t seq_len, hipStream_t stream) {
  if (!pool || seq_len < 0 || plane_stride <= 0) return TOPKV_ERR_INVALID_ARG;
  const topkv_launch_t l = {stream, nullptr, nullptr};
  const int64_t pages = pool->page_size > 0 ? ((int64_t)seq_len + pool->page_size - 1) / pool->page_size : 0;
  if (pages > INT32_MAX) return TOPKV_ERR_UNSUPPORTED;
  return topkv::launch_move(pack, pool, first_layer, packed, packed_cap, 1, block_table,
                            (int32_t)(pages > 0 ? pages : 1), nullptr, seq_len, 0, plane_stride, &l, layers,
                            layer_stride);
}

}  // namespace topkv_internal

// ---------------------------------------------------------------------------
// C ABI
// ---------------------------------------------------------------------------
extern "C" {

topkv_status_t topkv_pack_layer(const topkv_pool_t* src, int32_t layer, const int32_t* block_table,
                                int32_t seq_len, void* dst, hipStream_t stream) {
  if (!src || seq_len < 0) return TOPKV_ERR_INVALID_ARG;
  const topkv_launch_t l = {stream, nullptr, nullptr};
  const int64_t pages = src->page_size > 0 ? ((int64_t)seq_len + src->page_size - 1) / src->page_size : 0;
  const int64_t cap = topkv::single_bytes(src, seq_len);
  if (cap < 0 || pages > INT32_MAX) return TOPKV_ERR_UNSUPPORTED;
  return topkv::launch_move(true, src, layer, dst, cap, 1, block_table, (int32_t)(pages > 0 ? pages : 1),
                            nullptr, seq_len, 0, 0, &l);
}

topkv_status_t topkv_unpack_layer(const void* src, const topkv_pool_t* dst, int32_t layer,
                                  const int32_t* block_table, int32_t seq_len, hipStream_t stream) {
  if (!dst || seq_len < 0) return TOPKV_ERR_INVALID_ARG;
  const topkv_launch_t l = {stream, nullptr, nullptr};
  const int64_t pages = dst->page_size > 0 ? ((int64_t)seq_len + dst->page_size - 1) / dst->page_size : 0;
  const int64_t cap = topkv::single_bytes(dst, seq_len);
  if (cap < 0 || pages > INT32_MAX) return TOPKV_ERR_UNSUPPORTED;
  return topkv::launch_move(false, dst, layer, const_cast<void*>(src), cap, 1, block_table,
                            (int32_t)(pages > 0 ? pages : 1), nullptr, seq_len, 0, 0, &l);
}

topkv_status_t topkv_pack_layer_planes(const topkv_pool_t* src, int32_t layer, const int32_t* block_table,
                                       int32_t seq_len, void* dst, int64_t plane_stride, int64_t dst_bytes,
                                       hipStream_t stream) {
  if (!src || seq_len < 0 || plane_stride <= 0) return TOPKV_ERR_INVALID_ARG;
  const topkv_launch_t l = {stream, nullptr, nullptr};
  const int64_t pages = src->page_size > 0 ? ((int64_t)seq_len + src->page_size - 1) / src->page_size : 0;
  if (pages > INT32_MAX) return TOPKV_ERR_UNSUPPORTED;
  return topkv::launch_move(true, src, layer, dst, dst_bytes, 1, block_table, (int32_t)(pages > 0 ? pages : 1),
                            nullptr, seq_len, 0, plane_stride, &l);
}

topkv_status_t topkv_unpack_layer_planes(const void* src, int64_t plane_stride, int64_t src_bytes,
                                         const topkv_pool_t* dst, int32_t layer, const int32_t* block_table,
                                         int32_t seq_len, hipStream_t stream) {
  if (!dst || seq_len < 0 || plane_stride <= 0) return TOPKV_ERR_INVALID_ARG;
  const topkv_launch_t l = {stream, nullptr, nullptr};
  const int64_t pages = dst->page_size > 0 ? ((int64_t)seq_len + dst->page_size - 1) / dst->page_size : 0;
  if (pages > INT32_MAX) return TOPKV_ERR_UNSUPPORTED;
  return topkv::launch_move(false, dst, layer, const_cast<void*>(src), src_bytes, 1, block_table,
                            (int32_t)(pages > 0 ? pages : 1), nullptr, seq_len, 0, plane_stride, &l);
}

topkv_status_t topkv_pack_layer_window(const topkv_pool_t* src, int32_t layer, int32_t num_reqs,
                                       const int32_t* block_tables, int32_t bt_stride, const int32_t* seq_lens,
                                       int32_t window, void* dst, int64_t dst_bytes, const topkv_launch_t* launch) {
  if (num_reqs > 0 && !seq_lens) return TOPKV_ERR_INVALID_ARG;
  return topkv::launch_move(true, src, layer, dst, dst_bytes, num_reqs, block_tables, bt_stride,
                            num_reqs > 0 ? seq_lens : nullptr, 0, window, 0, launch);
}

topkv_status_t topkv_unpack_layer_window(const void* src, int64_t src_bytes, const topkv_pool_t* dst, int32_t layer,
                                         int32_t num_reqs, const int32_t* block_tables, int32_t bt_stride,
                                         const int32_t* seq_lens, int32_t window, const topkv_launch_t* launch) {
  if (num_reqs > 0 && !seq_lens) return TOPKV_ERR_INVALID_ARG;
  return topkv::launch_move(false, dst, layer, const_cast<void*>(src), src_bytes, num_reqs, block_tables,
                            bt_stride, num_reqs > 0 ? seq_lens : nullptr, 0, window, 0, launch);
}

topkv_status_t topkv_pack_layer_batched_ex(const topkv_pool_t* src, int32_t layer, int32_t num_reqs,
                                           const int32_t* block_tables, int32_t bt_stride,
                                           const int32_t* seq_lens, void* dst, int64_t dst_bytes,
                                           const topkv_launch_t* launch) {
  return topkv_pack_layer_window(src, layer, num_reqs, block_tables, bt_stride, seq_lens, 0, dst, dst_bytes,
                                 launch);
}

topkv_status_t topkv_unpack_layer_batched_ex(const void* src, int64_t src_bytes, const topkv_pool_t* dst,
                                             int32_t layer, int32_t num_reqs,
                                             const int32_t* block_tables, int32_t bt_stride,
                                             const int32_t* seq_lens, const topkv_launch_t* launch) {
  return topkv_unpack_layer_window(src, src_bytes, dst, layer, num_reqs, block_tables, bt_stride, seq_lens, 0,
                                   launch);
}

topkv_status_t topkv_pack_layer_batched(const topkv_pool_t* src, int32_t layer, int32_t num_reqs,
                                        const int32_t* block_tables, int32_t bt_stride,
                                        const int32_t* seq_lens, void* dst, int64_t dst_bytes,
                                        hipStream_t stream) {
  const topkv_launch_t l = {stream, nullptr, nullptr};
  return topkv_pack_layer_batched_ex(src, layer, num_reqs, block_tables, bt_stride, seq_lens, dst,
                                     dst_bytes, &l);
}

topkv_status_t topkv_unpack_layer_batched(const void* src, int64_t src_bytes, const topkv_pool_t* dst,
                                          int32_t layer, int32_t num_reqs, const int32_t* block_tables,
                                          int32_t bt_stride, const int32_t* seq_lens,
                                          hipStream_t stream) {
  const topkv_launch_t l = {stream, nullptr, nullptr};
  return topkv_unpack_layer_batched_ex(src, src_bytes, dst, layer, num_reqs, block_tables, bt_stride,
                                       seq_lens, &l);
}

int32_t topkv_engine_layers_per_grid(int32_t num_layers, int64_t layer_stride, const topkv_engine_t* engine) {
  if (num_layers < 1 || layer_stride < 0 || (engine && engine->layers_per_grid < 0)) return -1;
  return topkv::engine_layers_per_grid(num_layers, layer_stride, engine);
}

topkv_status_t topkv_engine_pack_layers(const topkv_pool_t* src, int32_t first_layer, int32_t num_layers,
                                        int32_t num_reqs, const int32_t* block_tables, int32_t bt_stride,
                                        const int32_t* seq_lens, void* packed, int64_t layer_stride,
                                        int64_t packed_bytes, const topkv_engine_t* engine, hipStream_t stream) {
  return topkv::engine_move(true, src, first_layer, num_layers, packed, packed_bytes, layer_stride, num_reqs,
                            block_tables, bt_stride, seq_lens, engine, stream);
}

topkv_status_t topkv_engine_unpack_layers(const void* packed, int64_t layer_stride, int64_t packed_bytes,
                                          const topkv_pool_t* dst, int32_t first_layer, int32_t num_layers,
                                          int32_t num_reqs, const int32_t* block_tables, int32_t bt_stride,
                                          const int32_t* seq_lens, const topkv_engine_t* engine,
                                          hipStream_t stream) {
  return topkv::engine_move(false, dst, first_layer, num_layers, const_cast<void*>(packed), packed_bytes,
                            layer_stride, num_reqs, block_tables, bt_stride, seq_lens, engine, stream);
}

int64_t topkv_packed_window_bytes(const topkv_pool_t* pool, const int32_t* seq_lens_host, int32_t num_reqs,
                                  int32_t window) {
  if (!pool || num_reqs < 0 || window < 0 || (num_reqs > 0 && !seq_lens_host)) return -1;
  if (pool->planes <= 0 || pool->num_heads <= 0 || pool->head_dim <= 0 || pool->elem_bytes <= 0) return -1;
  int64_t per_token;
  if (__builtin_mul_overflow((int64_t)pool->planes * pool->num_heads, (int64_t)pool->head_dim * pool->elem_bytes,
                             &per_token))
    return -1;
  int64_t total = 0;
  for (int32_t r = 0; r < num_reqs; ++r) {
    const int64_t n = seq_lens_host[r];
    if (n < 0) return -1;
    const int64_t kept = (window > 0 && n > window) ? window : n;
    int64_t b;
    if (__builtin_mul_overflow(per_token, kept, &b) || __builtin_add_overflow(total, b, &total)) return -1;
  }
  return total;
}

int64_t topkv_packed_layer_bytes(const topkv_pool_t* pool, const int32_t* seq_lens_host, int32_t num_reqs) {
  return topkv_packed_window_bytes(pool, seq_lens_host, num_reqs, 0);
}

const char* topkv_status_string(topkv_status_t status) {
  switch (status) {
    case TOPKV_OK: return "TOPKV_OK";
    case TOPKV_ERR_INVALID_ARG: return "TOPKV_ERR_INVALID_ARG: null pointer, bad layer or non-positive size";
    case TOPKV_ERR_UNSUPPORTED: return "TOPKV_ERR_UNSUPPORTED: size beyond the library's limits";
    case TOPKV_ERR_LAUNCH: return "TOPKV_ERR_LAUNCH: the HIP runtime refused the kernel launch";
    case TOPKV_ERR_BOUNDS: return "TOPKV_ERR_BOUNDS: block table entry, length, slot or packed capacity out of range";
    case TOPKV_ERR_DEVICE: return "TOPKV_ERR_DEVICE: HIP device query failed";
    case TOPKV_ERR_CHECKSUM: return "TOPKV_ERR_CHECKSUM: serialized header or checksum mismatch";
    case TOPKV_ERR_TIMEOUT: return "TOPKV_ERR_TIMEOUT: a layer's ready word did not arrive within the timeout";
    case TOPKV_ERR_CANCELLED: return "TOPKV_ERR_CANCELLED: the cancel word was set while a layer was awaited";
  }
  return "TOPKV_ERR_UNKNOWN";
}

}  // extern "C"
