// reshard.hip - one layer moved between cache layouts on gfx950: head-sliced
// pack and unpack (a tensor-parallel shard's heads), pool-to-pool
// re-blocking between page sizes without a staging buffer, and pools whose
// pages are head-major.  The layouts and the entry points are specified in
// include/topkv.h (per-layer unit: Section 5.2; K-then-V token-major wire
// order: Section 3.5; paged pools: Section 6; KV heads per layer: Sections
// 2.2 and 5.3).
//
// Design.  Every move copies, per request, kept token and plane, the moved
// heads' values.  The unit of contiguity is a granule: one head's head_dim
// values, or all moved heads at once when both sides keep heads adjacent (a
// packed buffer and a slot-major pool do, a head-major pool does not).  The
// work is flattened in the packed order (request, plane, token, granule,
// 16-byte piece), so
//   * a packed side's address is simply piece index * piece bytes, and both
//     sides walk consecutive bytes across consecutive lanes wherever their
//     layout allows (a head-major side still gets whole granules);
//   * the request comes from a binary search over per-request prefix sums
//     held in LDS (built with a wave64 shuffle scan from the device lengths),
//     every other index from multiply-high divisions by launch constants;
//   * when a token's pieces fill whole wave spans (every 70B-class shape),
//     request, plane, token and page are wave-uniform: they are computed once
//     per wave in scalar registers and the block-table entries come through
//     scalar loads, the last one reused while the page does not change.
// Granules are at least one head's values (256 bytes for head_dim 128 in
// bf16), so both sides touch whole cache lines: no LDS staging of the data is
// needed even where the layout transposes (slot-major <-> head-major).
// Each lane issues all of its loads before its stores; workgroups stride over
// tiles on a grid capped at a few workgroups per CU.  Table entries and
// lengths are bounds-checked on the device before any access.
#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>

#include <atomic>
#include <cstdint>

#include "internal.h"
#include "topkv.h"

namespace topkv_reshard {

#ifndef TOPKV_RS_VPT
#define TOPKV_RS_VPT 8            // pieces per lane per tile
#endif
#ifndef TOPKV_RS_SINGLE
#define TOPKV_RS_SINGLE 1         // direct grid for one request without a window
#endif
#ifndef TOPKV_RS_DIRECT
#define TOPKV_RS_DIRECT 1          // batches without a window take the direct grid when it fits
#endif
#ifndef TOPKV_XCD_REMAP
#define TOPKV_XCD_REMAP 0         // 1: each XCD takes a contiguous eighth of a direct grid (measured slower)
#endif
#ifndef TOPKV_EARLY_LENS
#define TOPKV_EARLY_LENS 1        // direct batches: earlier requests' lengths load with the request's own
#endif
#ifndef TOPKV_RS_WG_PER_CU
#define TOPKV_RS_WG_PER_CU 16     // grid cap = CUs * this
#endif

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kVpt = TOPKV_RS_VPT;
constexpr int kWgPerCu = TOPKV_RS_WG_PER_CU;

template <int B> struct Vec;
template <> struct Vec<16> { typedef unsigned int type __attribute__((ext_vector_type(4))); };
template <> struct Vec<8> { typedef unsigned int type __attribute__((ext_vector_type(2))); };
template <> struct Vec<4> { typedef unsigned int type; };
template <> struct Vec<2> { typedef unsigned short type; };
template <> struct Vec<1> { typedef unsigned char type; };

// n / d for 0 <= n < 2^31 by a multiply-high (Granlund and Montgomery, 1994):
// with s = ceil(log2 d) and m = floor(2^32 (2^s - d) / d) + 1, the quotient is
// (mulhi(n, m) + n) >> s; the sum cannot overflow because mulhi(n, m) <= n.
struct FastDiv {
  uint32_t d, m, s;
};

FastDiv make_div(uint32_t d) {
  uint32_t s = 0;
  while ((1ull << s) < d) ++s;
  const uint64_t m = (((1ull << 32) * ((1ull << s) - d)) / d) + 1;
  return FastDiv{d, (uint32_t)m, s};
}

__device__ __forceinline__ uint32_t fdiv(uint32_t n, const FastDiv& f) {
  return (__umulhi(n, f.m) + n) >> f.s;
}

// One side of a move (kernel argument, by value).
struct Side {
  char* base;               // pool: the layer slab; packed: the buffer
  int64_t layer_stride;     // several layers on grid z: bytes from one layer's base to the next
  const int32_t* tables;    // pool: [num_reqs][bt_stride]
  int64_t page_bytes;
  int64_t plane_bytes;
  int64_t head0_bytes;      // offset of the first moved head within a slot
  int64_t num_pages;        // valid page indices are [0, num_pages)
  int32_t slot_bytes;       // stride between slots of a page plane
  int32_t gran_stride;      // stride between consecutive granules of a slot
  int32_t bt_stride;
  int32_t packed;           // 1: packed buffer (shard regions of Params::packed_cap bytes)
  FastDiv page;             // tokens per page
};

struct Params {
  Side src, dst;
  int64_t packed_cap;       // bytes of each shard region of the packed side (one region unsharded)
  FastDiv vpg;              // pieces per granule
  FastDiv gpt;              // granules per (token, plane)
  FastDiv ktp;              // pieces per (token, plane) = gpt * vpg
  FastDiv gps;              // granules per shard (= gpt when unsharded)
  int32_t num_reqs;
  int32_t planes;
  int32_t window;
  int32_t max_tok;          // lengths are clamped to [0, max_tok]
  int32_t n_host;           // one request with a host-side length: its tokens (else unused)
  int32_t layers;           // direct grids: layers on grid z (1: one layer)
};

// Per-request kept-token counts and first kept tokens, and the exclusive
// prefix of planes * count (token-planes before request r), into LDS.
__device__ void request_prefix(const Params& p, const int32_t* __restrict__ seq_lens, int32_t* tp,
                               int32_t* st, int32_t* cnt, int32_t* wsum) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  int32_t carry = 0;
  for (int base = 0; base < p.num_reqs; base += kThreads) {
    const int r = base + threadIdx.x;
    int32_t v = 0;
    if (r < p.num_reqs) {
      int32_t n = seq_lens[r];
      n = n < 0 ? 0 : (n > p.max_tok ? p.max_tok : n);
      const int32_t start = (p.window > 0 && n > p.window) ? n - p.window : 0;
      st[r] = start;
      cnt[r] = n - start;
      v = (n - start) * p.planes;
    }
    int32_t x = v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int32_t y = __shfl_up(x, d, 64);
      if (lane >= d) x += y;
    }
    if (lane == 63) wsum[wave] = x;
    __syncthreads();
    int32_t before = carry, chunk = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      if (w < wave) before += wsum[w];
      chunk += wsum[w];
    }
    if (r < p.num_reqs) tp[r] = before + x - v;
    carry += chunk;
    __syncthreads();
  }
  if (threadIdx.x == 0) tp[p.num_reqs] = carry;
  __syncthreads();
}

// Byte offset of piece (r, c, t, k, e) on a pool side; false if the table
// entry is out of range.
__device__ __forceinline__ bool pool_offset(const Side& s, int32_t r, uint32_t c, uint32_t t, uint32_t k,
                                            uint32_t e_bytes, int64_t* off) {
  const uint32_t i = fdiv(t, s.page);
  const uint32_t slot = t - i * s.page.d;
  const int32_t page = s.tables[(int64_t)r * s.bt_stride + i];
  if (page < 0 || (int64_t)page >= s.num_pages) return false;
  *off = (int64_t)page * s.page_bytes + (int64_t)c * s.plane_bytes + (int64_t)slot * s.slot_bytes +
         s.head0_bytes + (int64_t)k * s.gran_stride + e_bytes;
  return true;
}

// Byte offset of piece (q2, k, e) on the packed side: granule k belongs to
// shard k / gps, which holds its own (request, plane, token)-ordered granules
// at shard * packed_cap.  Unsharded (gps = gpt) this is the piece index * VB.
// False past the shard's capacity.
template <int VB>
__device__ __forceinline__ bool packed_offset(const Params& p, uint32_t q2, uint32_t k, uint32_t e,
                                              int64_t* off) {
  const uint32_t sh = fdiv(k, p.gps);
  const uint32_t pos = k - sh * p.gps.d;
  const int64_t in_shard = ((int64_t)q2 * p.gps.d + pos) * ((int64_t)p.vpg.d * VB) + (int64_t)e * VB;
  *off = (int64_t)sh * p.packed_cap + in_shard;
  return in_shard + VB <= p.packed_cap;
}

struct Loc {
  int32_t r;                // request
  uint32_t c, t;            // plane, token
};

// Request, plane and token of global (request, plane, token) index q2: the
// largest r with tp[r] <= q2 owns it (its count is then > 0), and the plane
// is the number of whole token runs below q2 within the request.
__device__ __forceinline__ Loc locate(uint32_t q2, const int32_t* tp, const int32_t* st, const int32_t* cnt,
                                      int32_t num_reqs) {
  int lo = 0, hi = num_reqs - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if ((uint32_t)tp[mid] <= q2) lo = mid; else hi = mid - 1;
  }
  uint32_t local = q2 - (uint32_t)tp[lo];
  const uint32_t n_r = (uint32_t)cnt[lo];
  uint32_t c = 0;
  while (local >= n_r) { local -= n_r; ++c; }
  return Loc{lo, c, (uint32_t)st[lo] + local};
}

// Page lookups of one side for wave-uniform tokens.  Block tables are never
// written while a move runs, so they are read through the constant address
// space (scalar loads and the scalar cache); consecutive wave spans of a tile
// usually sit on the same page, so the last entry is kept.
struct PageCache {
  int32_t r = -1;
  uint32_t i = 0;
  int32_t page = -1;
};

typedef __attribute__((address_space(4))) const int32_t ConstInt;

// pool_offset for a wave-uniform (request, plane, token): the page lookup and
// everything but the piece's place inside the token's granules are uniform.
__device__ __forceinline__ bool pool_offset_wave(const Side& s, const Loc& at, uint32_t k, uint32_t e_bytes,
                                                 PageCache& pc, int64_t* off) {
  const uint32_t i = fdiv(at.t, s.page);
  const uint32_t slot = at.t - i * s.page.d;
  if (at.r != pc.r || i != pc.i) {
    const ConstInt* tab = (const ConstInt*)s.tables;
    pc.page = __builtin_amdgcn_readfirstlane(tab[(int64_t)at.r * s.bt_stride + i]);
    pc.r = at.r;
    pc.i = i;
  }
  const int32_t page = pc.page;
  if (page < 0 || (int64_t)page >= s.num_pages) return false;
  const int64_t base = (int64_t)page * s.page_bytes + (int64_t)at.c * s.plane_bytes +
                       (int64_t)slot * s.slot_bytes + s.head0_bytes;
  *off = base + (int64_t)k * s.gran_stride + e_bytes;
  return true;
}

// kWave: the pieces of one (request, plane, token) fill whole 64-piece wave
// spans (pieces per token-plane divisible by 64), so every wave instruction
// has one request, plane, token and page per side: those are found once per
// wave, with uniform (scalar) arithmetic and loads, and only the piece's
// place inside the token's granules varies across lanes.  Otherwise every
// lane locates its own piece.
template <int VB, bool kWave>
__global__ __launch_bounds__(kThreads) void kv_reshard_kernel(Params p, const int32_t* __restrict__ seq_lens) {
  typedef typename Vec<VB>::type V;
  extern __shared__ int32_t lds_i32[];
  int32_t* wsum = lds_i32;                     // [kWaves]
  int32_t* tp = wsum + kWaves;                 // [num_reqs + 1]
  int32_t* st = tp + (p.num_reqs + 1);         // [num_reqs]
  int32_t* cnt = st + p.num_reqs;              // [num_reqs]
  request_prefix(p, seq_lens, tp, st, cnt, wsum);

  const uint32_t per_tp = p.ktp.d;                            // pieces per (token, plane)
  const uint32_t total = (uint32_t)tp[p.num_reqs] * per_tp;   // the host keeps this below 2^31
  constexpr uint32_t kTile = (uint32_t)kThreads * kVpt;
  const uint32_t lane = threadIdx.x & 63u;
  const uint32_t wave_first = __builtin_amdgcn_readfirstlane(threadIdx.x & ~63u);

  PageCache src_pc, dst_pc;
  for (uint32_t base = blockIdx.x * kTile; base < total; base += gridDim.x * kTile) {
    // Three phases: every piece's addresses (searches, divisions, table
    // lookups), then every load, then every store.  No loop or branch sits
    // between the loads, so all kVpt of them are in flight at once; a skipped
    // piece loads from the source base (always valid) and is not stored.
    int64_t soff[kVpt], doff[kVpt];
    bool ok[kVpt];
#pragma unroll
    for (int j = 0; j < kVpt; ++j) {
      soff[j] = doff[j] = 0;
      ok[j] = false;
      if (kWave) {
        const uint32_t wbase = base + j * kThreads + wave_first;   // uniform
        if (wbase < total) {
          const uint32_t q2 = fdiv(wbase, p.ktp);
          const uint32_t m = wbase - q2 * per_tp + lane;            // < per_tp
          const uint32_t k = fdiv(m, p.vpg);
          const uint32_t e = m - k * p.vpg.d;
          Loc at = locate(q2, tp, st, cnt, p.num_reqs);
          at.r = __builtin_amdgcn_readfirstlane(at.r);
          at.c = __builtin_amdgcn_readfirstlane(at.c);
          at.t = __builtin_amdgcn_readfirstlane(at.t);
          int64_t so = 0, o = 0;
          // both sides' table entries are in-bounds reads whatever the other
          // side holds, so both lookups issue before either is tested
          const bool s_ok = p.src.packed ? packed_offset<VB>(p, q2, k, e, &so)
                                         : pool_offset_wave(p.src, at, k, e * VB, src_pc, &so);
          const bool d_ok = p.dst.packed ? packed_offset<VB>(p, q2, k, e, &o)
                                         : pool_offset_wave(p.dst, at, k, e * VB, dst_pc, &o);
          ok[j] = s_ok & d_ok;
          soff[j] = ok[j] ? so : 0;
          doff[j] = o;
        }
      } else {
        const uint32_t idx = base + j * kThreads + threadIdx.x;
        if (idx < total) {
          const uint32_t q = fdiv(idx, p.vpg);
          const uint32_t e = idx - q * p.vpg.d;
          const uint32_t q2 = fdiv(q, p.gpt);
          const uint32_t k = q - q2 * p.gpt.d;
          const Loc at = locate(q2, tp, st, cnt, p.num_reqs);
          int64_t so = 0, o = 0;
          const bool s_ok = p.src.packed ? packed_offset<VB>(p, q2, k, e, &so)
                                         : pool_offset(p.src, at.r, at.c, at.t, k, e * VB, &so);
          const bool d_ok = p.dst.packed ? packed_offset<VB>(p, q2, k, e, &o)
                                         : pool_offset(p.dst, at.r, at.c, at.t, k, e * VB, &o);
          ok[j] = s_ok & d_ok;
          soff[j] = ok[j] ? so : 0;
          doff[j] = o;
        }
      }
    }
    V v[kVpt];
#pragma unroll
    for (int j = 0; j < kVpt; ++j) v[j] = __builtin_nontemporal_load(reinterpret_cast<const V*>(p.src.base + soff[j]));
#pragma unroll
    for (int j = 0; j < kVpt; ++j)
      if (ok[j]) __builtin_nontemporal_store(v[j], reinterpret_cast<V*>(p.dst.base + doff[j]));
  }
}

// Kept tokens (window 0) of requests [0, r): the (plane, token) offset of
// request r in the packed order is planes times this.  Each wave sums the
// lengths on its own (lanes stride over them, then a butterfly), so no LDS and
// no barrier are involved.
// `mine` is seq_lens[lane] for lanes below r, already loaded by the caller.
__device__ __forceinline__ int32_t kept_before(const int32_t* __restrict__ seq_lens, int32_t r, int32_t max_tok,
                                               int32_t mine) {
  const int lane = threadIdx.x & 63;
  int32_t s = 0;
  for (int j = lane; j < r; j += 64) {
    int32_t n = j == lane ? mine : seq_lens[j];
    s += n < 0 ? 0 : (n > max_tok ? max_tok : n);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
  return __builtin_amdgcn_readfirstlane(s);
}

// Direct grid without a window, wave-uniform tokens (every 70B-class shape):
// workgroup (x, y[, z]) copies tile x of plane y [of request z], in packed
// order.  A token's page depends only on the token, not on the request's
// length, so each wave's first page lookups go out together with the length
// load; there is no prefix scan.  Pieces of tokens at or past the (clamped)
// length are skipped.  kBatch: requests on grid z, each at the (plane, token)
// offset of the lengths before it, and tiles past a request's length exit at
// once; otherwise one request.  kHostLen: the one request's length is the
// launch constant n_host instead of a device value.
// Workgroup coordinates of a direct grid.  The dispatcher hands linear
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

template <int VB, bool kBatch, bool kHostLen = false>
__device__ __forceinline__ void direct_move(const Params& p, const int32_t* __restrict__ seq_lens) {
  typedef typename Vec<VB>::type V;
  constexpr uint32_t kTile = (uint32_t)kThreads * kVpt;
  const uint32_t per_tp = p.ktp.d;
  const uint32_t lane = threadIdx.x & 63u;
  const uint32_t wave_first = __builtin_amdgcn_readfirstlane(threadIdx.x & ~63u);
  const uint3 b = grid_block();
  const uint32_t c = b.y;
  // grid z: the layer (one request), or layer * num_reqs + request (a batch over several layers)
  uint32_t lz = 0;
  int32_t r = 0;
  if (!kBatch) {
    lz = b.z;
  } else if (p.layers > 1) {
    lz = b.z / (uint32_t)p.num_reqs;
    r = (int32_t)(b.z - lz * (uint32_t)p.num_reqs);
  } else {
    r = (int32_t)b.z;
  }
  const char* const src_base = p.src.base + (int64_t)lz * p.src.layer_stride;
  char* const dst_base = p.dst.base + (int64_t)lz * p.dst.layer_stride;
  const uint32_t base = b.x * kTile;
  PageCache src_pc, dst_pc;
  {
    // the first span's token is known before the length: prime the page caches
    const uint32_t t0 = fdiv(base + wave_first, p.ktp);
    if (t0 < (uint32_t)p.max_tok) {
      const Loc at0{r, c, t0};
      int64_t unused;
      if (!p.src.packed) pool_offset_wave(p.src, at0, 0, 0, src_pc, &unused);
      if (!p.dst.packed) pool_offset_wave(p.dst, at0, 0, 0, dst_pc, &unused);
    }
  }
  // with a batch, each lane below r also loads one earlier request's length
  // (for the request's packed offset) next to this request's own
  int32_t mine = 0;
#if TOPKV_EARLY_LENS
  if (kBatch && (int32_t)lane < r) mine = __builtin_nontemporal_load(seq_lens + lane);
#endif
  int32_t n = kHostLen ? p.n_host : __builtin_amdgcn_readfirstlane(seq_lens[r]);
#if TOPKV_EARLY_LENS
  if (kBatch) asm volatile("" ::"v"(mine));   // keep the load here: not sunk past the exit test below
#else
  if (kBatch && (int32_t)lane < r) mine = seq_lens[lane];
#endif
  n = n < 0 ? 0 : (n > p.max_tok ? p.max_tok : n);
  const uint32_t end = (uint32_t)n * per_tp;                  // pieces of this plane
  if (kBatch && base >= end) return;                          // past this request's tokens
  const uint32_t q0 = (kBatch && r > 0) ? (uint32_t)(p.planes * kept_before(seq_lens, r, p.max_tok, mine)) : 0u;
  // Each load issues as soon as its address is known (there is no loop here
  // to hold it up); a skipped piece loads the source base and is not stored.
  V v[kVpt];
  int64_t doff[kVpt];
  bool ok[kVpt];
#pragma unroll
  for (int j = 0; j < kVpt; ++j) {
    int64_t soff = 0;
    doff[j] = 0;
    ok[j] = false;
    const uint32_t wbase = base + j * kThreads + wave_first;    // uniform, within plane c
    if (wbase < end) {
      const uint32_t t = fdiv(wbase, p.ktp);
      const uint32_t m = wbase - t * per_tp + lane;
      const uint32_t k = fdiv(m, p.vpg);
      const uint32_t e = m - k * p.vpg.d;
      const Loc at{r, c, t};
      const uint32_t q2 = q0 + c * (uint32_t)n + t;             // global (request, plane, token) index
      int64_t so = 0, o = 0;
      const bool s_ok = p.src.packed ? packed_offset<VB>(p, q2, k, e, &so)
                                     : pool_offset_wave(p.src, at, k, e * VB, src_pc, &so);
      const bool d_ok = p.dst.packed ? packed_offset<VB>(p, q2, k, e, &o)
                                     : pool_offset_wave(p.dst, at, k, e * VB, dst_pc, &o);
      ok[j] = s_ok & d_ok;
      soff = ok[j] ? so : 0;
      doff[j] = o;
    }
    v[j] = __builtin_nontemporal_load(reinterpret_cast<const V*>(src_base + soff));
  }
#pragma unroll
  for (int j = 0; j < kVpt; ++j)
    if (ok[j]) __builtin_nontemporal_store(v[j], reinterpret_cast<V*>(dst_base + doff[j]));
}

template <int VB, bool kHostLen>
__global__ __launch_bounds__(kThreads) void kv_reshard_single_kernel(Params p,
                                                                    const int32_t* __restrict__ seq_lens) {
  direct_move<VB, false, kHostLen>(p, seq_lens);
}

template <int VB>
__global__ __launch_bounds__(kThreads) void kv_reshard_direct_kernel(Params p,
                                                                    const int32_t* __restrict__ seq_lens) {
  direct_move<VB, true>(p, seq_lens);
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------

constexpr int kMaxDevices = 64;
std::atomic<int> g_cus[kMaxDevices];

topkv_status_t cu_count(int* out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return TOPKV_ERR_DEVICE;
  const int cached = dev < kMaxDevices ? g_cus[dev].load(std::memory_order_relaxed) : 0;
  if (cached > 0) { *out = cached; return TOPKV_OK; }
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    return TOPKV_ERR_DEVICE;
  if (dev < kMaxDevices) g_cus[dev].store(cus, std::memory_order_relaxed);
  *out = cus;
  return TOPKV_OK;
}

struct PoolInfo {
  int64_t head_bytes, slot_bytes, plane_bytes, page_bytes, layer_bytes;
};

// Strides of a pool view in its layout, after validating the descriptor.
topkv_status_t pool_info(const topkv_view_t* v, int32_t head_count, PoolInfo* g) {
  const topkv_pool_t& pl = v->pool;
  if (!pl.base || pl.num_pages <= 0 || pl.num_layers <= 0 || pl.page_size <= 0 || pl.planes <= 0 ||
      pl.num_heads <= 0 || pl.head_dim <= 0)
    return TOPKV_ERR_INVALID_ARG;
  if (pl.elem_bytes != 1 && pl.elem_bytes != 2 && pl.elem_bytes != 4 && pl.elem_bytes != 8)
    return TOPKV_ERR_INVALID_ARG;
  if (v->layer < 0 || v->layer >= pl.num_layers || v->bt_stride <= 0 || v->head_begin < 0 ||
      head_count > pl.num_heads - v->head_begin)
    return TOPKV_ERR_INVALID_ARG;
  int64_t head, row, plane, page, layer, all;
  if (__builtin_mul_overflow((int64_t)pl.head_dim, (int64_t)pl.elem_bytes, &head) ||
      __builtin_mul_overflow(head, (int64_t)pl.num_heads, &row) ||
      __builtin_mul_overflow(row, (int64_t)pl.page_size, &plane) ||
      __builtin_mul_overflow(plane, (int64_t)pl.planes, &page) ||
      __builtin_mul_overflow(page, pl.num_pages, &layer) ||
      __builtin_mul_overflow(layer, (int64_t)pl.num_layers, &all))
    return TOPKV_ERR_UNSUPPORTED;
  if (plane > INT32_MAX || pl.num_pages > INT32_MAX) return TOPKV_ERR_UNSUPPORTED;
  const bool head_major = v->layout == TOPKV_LAYOUT_POOL_HEAD_MAJOR;
  g->head_bytes = head_major ? head * pl.page_size : head;
  g->slot_bytes = head_major ? head : row;
  g->plane_bytes = plane;
  g->page_bytes = page;
  g->layer_bytes = layer;
  return TOPKV_OK;
}

bool valid_layout(int32_t l) {
  return l == TOPKV_LAYOUT_PACKED || l == TOPKV_LAYOUT_POOL || l == TOPKV_LAYOUT_POOL_HEAD_MAJOR;
}

typedef void (*KernelFn)(Params, const int32_t*);

template <bool kWave>
KernelFn kernel_for_mode(int vb) {
  switch (vb) {
    case 16: return kv_reshard_kernel<16, kWave>;
    case 8: return kv_reshard_kernel<8, kWave>;
    case 4: return kv_reshard_kernel<4, kWave>;
    case 2: return kv_reshard_kernel<2, kWave>;
    default: return kv_reshard_kernel<1, kWave>;
  }
}

KernelFn kernel_for(int vb, bool wave) { return wave ? kernel_for_mode<true>(vb) : kernel_for_mode<false>(vb); }

template <bool kHostLen>
KernelFn single_kernel_for(int vb) {
  switch (vb) {
    case 16: return kv_reshard_single_kernel<16, kHostLen>;
    case 8: return kv_reshard_single_kernel<8, kHostLen>;
    case 4: return kv_reshard_single_kernel<4, kHostLen>;
    case 2: return kv_reshard_single_kernel<2, kHostLen>;
    default: return kv_reshard_single_kernel<1, kHostLen>;
  }
}

KernelFn direct_kernel_for(int vb) {
  switch (vb) {
    case 16: return kv_reshard_direct_kernel<16>;
    case 8: return kv_reshard_direct_kernel<8>;
    case 4: return kv_reshard_direct_kernel<4>;
    case 2: return kv_reshard_direct_kernel<2>;
    default: return kv_reshard_direct_kernel<1>;
  }
}

// single_only: launch only the one-request direct grid (and report whether it
// did through *launched); otherwise whichever grid applies.  layers > 1: the
// views' layers and the next layers - 1 on grid z of a direct grid (a pool
// side's layer slabs follow each other; a packed side's layer z starts at
// data + z * packed_layer_stride), launched only when a direct grid applies:
// *launched stays false otherwise, with nothing queued.  The caller has
// checked the layer ranges and the stride.
topkv_status_t move_layer_impl(const topkv_view_t* src, const topkv_view_t* dst, int32_t num_reqs,
                               const int32_t* seq_lens, int32_t head_count, int32_t window,
                               const topkv_launch_t& launch, bool single_only, bool* launched,
                               int32_t n_host = -1, int32_t layers = 1, int64_t packed_layer_stride = 0) {
  *launched = false;
  if (!src || !dst || !valid_layout(src->layout) || !valid_layout(dst->layout)) return TOPKV_ERR_INVALID_ARG;
  if (src->layout == TOPKV_LAYOUT_PACKED && dst->layout == TOPKV_LAYOUT_PACKED) return TOPKV_ERR_INVALID_ARG;
  // a host-side length (n_host >= 0) stands for seq_lens: one request, one-request grid only
  const bool host_len = n_host >= 0;
  if (host_len && (num_reqs != 1 || !single_only || seq_lens)) return TOPKV_ERR_INVALID_ARG;
  if (num_reqs < 0 || head_count <= 0 || window < 0 || (num_reqs > 0 && !seq_lens && !host_len))
    return TOPKV_ERR_INVALID_ARG;
  if (num_reqs > TOPKV_MAX_BATCH_REQS) return TOPKV_ERR_UNSUPPORTED;

  const topkv_view_t* sides[2] = {src, dst};
  const topkv_pool_t* geo = nullptr;     // geometry both pool sides share
  PoolInfo info[2] = {};
  int64_t packed_cap = 0;
  int64_t shards = 1;
  int64_t max_tok = INT32_MAX;
  for (int i = 0; i < 2; ++i) {
    const topkv_view_t* v = sides[i];
    if (v->layout == TOPKV_LAYOUT_PACKED) {
      if (v->bytes < 0 || (v->bytes > 0 && !v->data) || v->shards < 0) return TOPKV_ERR_INVALID_ARG;
      packed_cap = v->bytes;
      shards = v->shards > 1 ? v->shards : 1;
      if (head_count % shards != 0) return TOPKV_ERR_INVALID_ARG;
      continue;
    }
    const topkv_status_t st = pool_info(v, head_count, &info[i]);
    if (st != TOPKV_OK) return st;
    if (num_reqs > 0 && !v->block_tables) return TOPKV_ERR_INVALID_ARG;
    if (geo && (geo->planes != v->pool.planes || geo->head_dim != v->pool.head_dim ||
                geo->elem_bytes != v->pool.elem_bytes))
      return TOPKV_ERR_INVALID_ARG;
    geo = &v->pool;
    const int64_t cap = (int64_t)v->bt_stride * v->pool.page_size;
    if (cap < max_tok) max_tok = cap;
  }
  if (num_reqs == 0) return TOPKV_OK;

  // Checked mode: validate each pool side's tables (an unpack destination for
  // pages named twice), and the packed side's room for every kept token.  The
  // one-request route from a pack/unpack call was checked by its caller.
  if (!single_only && topkv_internal::checked_mode()) {
    const bool has_packed = src->layout == TOPKV_LAYOUT_PACKED || dst->layout == TOPKV_LAYOUT_PACKED;
    const int64_t per_token = (int64_t)geo->planes * (head_count / shards) * geo->head_dim * geo->elem_bytes;
    bool cap_checked = false;
    for (int i = 0; i < 2; ++i) {
      const topkv_view_t* v = sides[i];
      if (v->layout == TOPKV_LAYOUT_PACKED) continue;
      const bool with_cap = has_packed && !cap_checked;
      const topkv_status_t cs = topkv_internal::checked_tables(
          &v->pool, num_reqs, v->block_tables, v->bt_stride, seq_lens, 0, window, i == 1, with_cap ? per_token : 0,
          0, with_cap ? packed_cap : INT64_MAX, launch.stream);
      if (cs != TOPKV_OK) return cs;
      cap_checked = cap_checked || with_cap;
    }
  }

  // Heads ride together in one granule when both sides keep them adjacent.
  const int64_t head = (int64_t)geo->head_dim * geo->elem_bytes;
  bool adjacent = true;
  for (int i = 0; i < 2; ++i)
    if (sides[i]->layout == TOPKV_LAYOUT_POOL_HEAD_MAJOR) adjacent = false;
  const int64_t heads_per_gran = adjacent ? head_count / shards : 1;
  const int64_t gran = heads_per_gran * head;
  // Piece width: every stride and base the pieces are addressed with.
  int vb = 16;
  for (; vb > 1; vb >>= 1) {
    bool fits = gran % vb == 0;
    for (int i = 0; i < 2 && fits; ++i) {
      const topkv_view_t* v = sides[i];
      if (v->layout == TOPKV_LAYOUT_PACKED) {
        fits = reinterpret_cast<uintptr_t>(v->data) % vb == 0 && (shards == 1 || packed_cap % vb == 0) &&
               packed_layer_stride % vb == 0;
      } else {
        const uintptr_t b = reinterpret_cast<uintptr_t>(v->pool.base);
        fits = b % vb == 0 && info[i].layer_bytes % vb == 0 && info[i].page_bytes % vb == 0 &&
               info[i].plane_bytes % vb == 0 && info[i].slot_bytes % vb == 0 && info[i].head_bytes % vb == 0;
      }
    }
    if (fits) break;
  }
  const int64_t vpg = gran / vb;
  const int64_t gpt = head_count / heads_per_gran;
  // Upper bound of pieces in the launch; indices are 32-bit in the kernel.
  if (max_tok <= 0) return TOPKV_OK;
  int64_t bound;
  if (__builtin_mul_overflow((int64_t)num_reqs * max_tok, (int64_t)geo->planes, &bound) ||
      __builtin_mul_overflow(bound, gpt * vpg, &bound) || bound >= ((int64_t)1 << 31) || vpg >= ((int64_t)1 << 31))
    return TOPKV_ERR_UNSUPPORTED;
  // Skipped pieces load from the source's base, so it must hold one piece; a
  // packed source smaller than that holds nothing to move.
  if (src->layout == TOPKV_LAYOUT_PACKED && packed_cap < vb) return TOPKV_OK;

  Params p = {};
  for (int i = 0; i < 2; ++i) {
    const topkv_view_t* v = sides[i];
    Side& s = i == 0 ? p.src : p.dst;
    if (v->layout == TOPKV_LAYOUT_PACKED) {
      s.base = static_cast<char*>(v->data);
      s.layer_stride = packed_layer_stride;
      s.packed = 1;
      s.page = make_div(1);
      continue;
    }
    s.base = static_cast<char*>(v->pool.base) + (int64_t)v->layer * info[i].layer_bytes;
    s.layer_stride = info[i].layer_bytes;
    s.tables = v->block_tables;
    s.page_bytes = info[i].page_bytes;
    s.plane_bytes = info[i].plane_bytes;
    s.head0_bytes = (int64_t)v->head_begin * info[i].head_bytes;
    s.num_pages = v->pool.num_pages;
    s.slot_bytes = (int32_t)info[i].slot_bytes;
    s.gran_stride = (int32_t)(heads_per_gran * info[i].head_bytes);
    s.bt_stride = v->bt_stride;
    s.page = make_div((uint32_t)v->pool.page_size);
  }
  p.packed_cap = packed_cap;
  p.vpg = make_div((uint32_t)vpg);
  p.gpt = make_div((uint32_t)gpt);
  p.ktp = make_div((uint32_t)(gpt * vpg));
  p.gps = make_div((uint32_t)(gpt / shards));
  p.num_reqs = num_reqs;
  p.planes = geo->planes;
  p.window = window;
  p.max_tok = (int32_t)max_tok;
  p.n_host = host_len ? (n_host < max_tok ? n_host : (int32_t)max_tok) : 0;
  p.layers = layers;

  int cus = 0;
  const topkv_status_t st = cu_count(&cus);
  if (st != TOPKV_OK) return st;
  const int64_t tile = (int64_t)kThreads * kVpt;
  int64_t blocks = (bound + tile - 1) / tile;
  if (blocks > (int64_t)cus * kWgPerCu) blocks = (int64_t)cus * kWgPerCu;
  if (blocks < 1) blocks = 1;
  const size_t lds = sizeof(int32_t) * (kWaves + 3 * (size_t)num_reqs + 1);
  const bool wave = (gpt * vpg) % 64 == 0;
  // a host-side length sizes the grid exactly; a device one by the table's capacity
  const int64_t grid_tok = host_len ? p.n_host : max_tok;
  const int64_t plane_tiles = (grid_tok * gpt * vpg + tile - 1) / tile;
  const bool single = TOPKV_RS_SINGLE && num_reqs == 1 && window == 0 && wave && plane_tiles <= INT32_MAX &&
                      geo->planes <= 65535;
  // a batch without a window: the same direct grid with requests on z, while it stays within
  // 2^20 workgroups and 1024 requests (each workgroup sums the lengths before its request)
  const bool direct = !single && TOPKV_RS_DIRECT && num_reqs > 1 && num_reqs <= 1024 && window == 0 && wave &&
                      geo->planes <= 65535 && plane_tiles * geo->planes * num_reqs <= ((int64_t)1 << 20);
  if (single_only && !single) return TOPKV_OK;
  if (layers > 1 && !((single && layers <= 65535) || (direct && (int64_t)num_reqs * layers <= 65535))) return TOPKV_OK;
  const dim3 grid = single   ? dim3((unsigned)plane_tiles, (unsigned)geo->planes, (unsigned)layers)
                    : direct ? dim3((unsigned)plane_tiles, (unsigned)geo->planes, (unsigned)(num_reqs * layers))
                             : dim3((unsigned)blocks);
  if (plane_tiles == 0) return TOPKV_OK;   // a host-side length of 0: nothing to move
  const KernelFn fn = single   ? (host_len ? single_kernel_for<true>(vb) : single_kernel_for<false>(vb))
                      : direct ? direct_kernel_for(vb)
                               : kernel_for(vb, wave);
  const size_t shmem = (single || direct) ? 0 : lds;
  if (launch.start || launch.stop)
    hipExtLaunchKernelGGL(fn, grid, dim3(kThreads), shmem, launch.stream, launch.start, launch.stop, 0, p, seq_lens);
  else
    hipLaunchKernelGGL(fn, grid, dim3(kThreads), shmem, launch.stream, p, seq_lens);
  if (hipGetLastError() != hipSuccess) return TOPKV_ERR_LAUNCH;
  *launched = true;
  return TOPKV_OK;
}

topkv_status_t move_layer(const topkv_view_t* src, const topkv_view_t* dst, int32_t num_reqs,
                          const int32_t* seq_lens, int32_t head_count, int32_t window, hipStream_t stream) {
  topkv_launch_t launch = {stream, nullptr, nullptr};
  bool launched = false;
  return move_layer_impl(src, dst, num_reqs, seq_lens, head_count, window, launch, false, &launched);
}

// Layers [view.layer, view.layer + num_layers) of each pool side (a packed
// side's layer z at data + z * packed_layer_stride), in grids of
// topkv_engine_layers_per_grid layers (the bytes a layer moves: the packed
// side's regions, or for pool to pool the source tables' capacity); a move
// no direct grid takes runs one launch per layer.
topkv_status_t move_layers(const topkv_view_t* src, const topkv_view_t* dst, int32_t num_layers,
                           int64_t packed_layer_stride, int32_t num_reqs, const int32_t* seq_lens,
                           int32_t head_count, int32_t window, hipStream_t stream) {
  if (!src || !dst || num_layers < 0 || packed_layer_stride < 0 || head_count <= 0) return TOPKV_ERR_INVALID_ARG;
  if (!valid_layout(src->layout) || !valid_layout(dst->layout)) return TOPKV_ERR_INVALID_ARG;
  const topkv_view_t* sides[2] = {src, dst};
  int64_t layer_bytes = 0;   // bytes one layer moves, at most (sizes the grids only)
  for (int i = 0; i < 2; ++i) {
    const topkv_view_t* v = sides[i];
    if (v->layout == TOPKV_LAYOUT_PACKED) {
      const int64_t regions = v->shards > 1 ? v->shards : 1;
      int64_t span;
      if (v->bytes < 0 || v->shards < 0 || __builtin_mul_overflow(regions, v->bytes, &span))
        return TOPKV_ERR_INVALID_ARG;
      if (num_layers > 1 && packed_layer_stride < span) return TOPKV_ERR_INVALID_ARG;   // layers would overlap
      layer_bytes = span;
      continue;
    }
    if (v->layer < 0 || num_layers > v->pool.num_layers - v->layer) return TOPKV_ERR_INVALID_ARG;
  }
  int64_t last;   // the last layer's offset on a packed side
  if (num_layers > 1 && __builtin_mul_overflow((int64_t)(num_layers - 1), packed_layer_stride, &last))
    return TOPKV_ERR_INVALID_ARG;
  if (num_layers == 0 || num_reqs == 0) return TOPKV_OK;
  if (layer_bytes == 0) {   // pool to pool: the source tables' capacity in tokens, every moved head
    const topkv_pool_t& g = src->pool;
    const int64_t factors[] = {src->bt_stride, g.page_size, g.planes, head_count, g.head_dim, g.elem_bytes};
    layer_bytes = num_reqs;
    for (const int64_t f : factors)
      if (f < 0 || __builtin_mul_overflow(layer_bytes, f, &layer_bytes)) {
        layer_bytes = INT64_MAX;   // only sizes the grids; the move itself validates the pool
        break;
      }
  }
  const int32_t per = topkv_engine_layers_per_grid(num_layers, layer_bytes, nullptr);
  if (per < 1) return TOPKV_ERR_INVALID_ARG;
  topkv_launch_t launch = {stream, nullptr, nullptr};
  for (int32_t j = 0; j < num_layers; j += per) {
    const int32_t n = num_layers - j < per ? num_layers - j : per;
    topkv_view_t s = *src, d = *dst;
    topkv_view_t* moved[2] = {&s, &d};
    for (topkv_view_t* v : moved) {
      if (v->layout == TOPKV_LAYOUT_PACKED)
        v->data = v->data ? static_cast<char*>(v->data) + (int64_t)j * packed_layer_stride : nullptr;
      else
        v->layer += j;
    }
    bool launched = false;
    topkv_status_t st = n > 1 ? move_layer_impl(&s, &d, num_reqs, seq_lens, head_count, window, launch, false,
                                                &launched, -1, n, packed_layer_stride)
                              : TOPKV_OK;
    if (st != TOPKV_OK) return st;
    if (launched) continue;
    // one launch per layer (one layer in this group, or a move no direct grid takes)
    for (int32_t l = 0; l < n; ++l) {
      topkv_view_t s1 = s, d1 = d;
      topkv_view_t* one[2] = {&s1, &d1};
      for (topkv_view_t* v : one) {
        if (v->layout == TOPKV_LAYOUT_PACKED)
          v->data = v->data ? static_cast<char*>(v->data) + (int64_t)l * packed_layer_stride : nullptr;
        else
          v->layer += l;
      }
      st = move_layer_impl(&s1, &d1, num_reqs, seq_lens, head_count, window, launch, false, &launched);
      if (st != TOPKV_OK) return st;
    }
  }
  return TOPKV_OK;
}

topkv_view_t pool_view(int32_t layout, const topkv_pool_t* pool, int32_t layer, const int32_t* tables,
                       int32_t bt_stride, int32_t head_begin) {
  topkv_view_t v = {};
  v.layout = layout;
  v.layer = layer;
  v.head_begin = head_begin;
  v.bt_stride = bt_stride;
  v.block_tables = tables;
  v.pool = *pool;
  return v;
}

topkv_view_t packed_view(const void* data, int64_t bytes, int32_t shards = 1) {
  topkv_view_t v = {};
  v.layout = TOPKV_LAYOUT_PACKED;
  v.data = const_cast<void*>(data);
  v.bytes = bytes;
  v.shards = shards;
  return v;
}

}  // namespace topkv_reshard

using namespace topkv_reshard;

namespace topkv_internal {

topkv_status_t single_request_move(bool pack, const topkv_pool_t* pool, int32_t layer, void* packed,
                                   int64_t packed_cap, const int32_t* tables, int32_t bt_stride,
                                   const int32_t* seq_lens, int32_t seq_len, const topkv_launch_t* launch,
                                   bool* launched) {
  *launched = false;
  const topkv_view_t pv = pool_view(TOPKV_LAYOUT_POOL, pool, layer, tables, bt_stride, 0);
  const topkv_view_t kv = packed_view(packed, packed_cap, 1);
  const int32_t n_host = seq_lens ? -1 : seq_len;
  const topkv_status_t st =
      pack ? move_layer_impl(&pv, &kv, 1, seq_lens, pool->num_heads, 0, *launch, true, launched, n_host)
           : move_layer_impl(&kv, &pv, 1, seq_lens, pool->num_heads, 0, *launch, true, launched, n_host);
  // anything this path does not take (limits, shapes) goes back to the caller's kernel
  if (st == TOPKV_ERR_INVALID_ARG || st == TOPKV_ERR_UNSUPPORTED || st == TOPKV_ERR_BOUNDS) {
    *launched = false;
    return TOPKV_OK;
  }
  return st;
}

}  // namespace topkv_internal

extern "C" {

topkv_status_t topkv_move_layer(const topkv_view_t* src, const topkv_view_t* dst, int32_t num_reqs,
                                const int32_t* seq_lens, int32_t head_count, int32_t window,
                                hipStream_t stream) {
  return move_layer(src, dst, num_reqs, seq_lens, head_count, window, stream);
}

topkv_status_t topkv_move_layers(const topkv_view_t* src, const topkv_view_t* dst, int32_t num_layers,
                                 int64_t packed_layer_stride, int32_t num_reqs, const int32_t* seq_lens,
                                 int32_t head_count, int32_t window, hipStream_t stream) {
  return move_layers(src, dst, num_layers, packed_layer_stride, num_reqs, seq_lens, head_count, window, stream);
}

topkv_status_t topkv_pack_layer_heads(const topkv_pool_t* src, int32_t layer, int32_t num_reqs,
                                      const int32_t* block_tables, int32_t bt_stride, const int32_t* seq_lens,
                                      int32_t head_begin, int32_t head_count, void* dst, int64_t dst_bytes,
                                      hipStream_t stream) {
  if (!src) return TOPKV_ERR_INVALID_ARG;
  const topkv_view_t s = pool_view(TOPKV_LAYOUT_POOL, src, layer, block_tables, bt_stride, head_begin);
  const topkv_view_t d = packed_view(dst, dst_bytes);
  return move_layer(&s, &d, num_reqs, seq_lens, head_count, 0, stream);
}

topkv_status_t topkv_unpack_layer_heads(const void* src, int64_t src_bytes, const topkv_pool_t* dst,
                                        int32_t layer, int32_t num_reqs, const int32_t* block_tables,
                                        int32_t bt_stride, const int32_t* seq_lens, int32_t head_begin,
                                        int32_t head_count, hipStream_t stream) {
  if (!dst) return TOPKV_ERR_INVALID_ARG;
  const topkv_view_t s = packed_view(src, src_bytes);
  const topkv_view_t d = pool_view(TOPKV_LAYOUT_POOL, dst, layer, block_tables, bt_stride, head_begin);
  return move_layer(&s, &d, num_reqs, seq_lens, head_count, 0, stream);
}

topkv_status_t topkv_pack_layer_shards(const topkv_pool_t* src, int32_t layer, int32_t num_reqs,
                                      const int32_t* block_tables, int32_t bt_stride, const int32_t* seq_lens,
                                      int32_t head_begin, int32_t head_count, int32_t shards, void* dst,
                                      int64_t shard_bytes, hipStream_t stream) {
  if (!src || shards < 1) return TOPKV_ERR_INVALID_ARG;
  const topkv_view_t s = pool_view(TOPKV_LAYOUT_POOL, src, layer, block_tables, bt_stride, head_begin);
  const topkv_view_t d = packed_view(dst, shard_bytes, shards);
  return move_layer(&s, &d, num_reqs, seq_lens, head_count, 0, stream);
}

topkv_status_t topkv_unpack_layer_shards(const void* src, int64_t shard_bytes, int32_t shards,
                                        const topkv_pool_t* dst, int32_t layer, int32_t num_reqs,
                                        const int32_t* block_tables, int32_t bt_stride, const int32_t* seq_lens,
                                        int32_t head_begin, int32_t head_count, hipStream_t stream) {
  if (!dst || shards < 1) return TOPKV_ERR_INVALID_ARG;
  const topkv_view_t s = packed_view(src, shard_bytes, shards);
  const topkv_view_t d = pool_view(TOPKV_LAYOUT_POOL, dst, layer, block_tables, bt_stride, head_begin);
  return move_layer(&s, &d, num_reqs, seq_lens, head_count, 0, stream);
}

topkv_status_t topkv_reblock_layer(const topkv_pool_t* src, int32_t src_layer, const int32_t* src_tables,
                                   int32_t src_stride, const topkv_pool_t* dst, int32_t dst_layer,
                                   const int32_t* dst_tables, int32_t dst_stride, int32_t num_reqs,
                                   const int32_t* seq_lens, hipStream_t stream) {
  if (!src || !dst) return TOPKV_ERR_INVALID_ARG;
  if (src->num_heads != dst->num_heads) return TOPKV_ERR_INVALID_ARG;
  const topkv_view_t s = pool_view(TOPKV_LAYOUT_POOL, src, src_layer, src_tables, src_stride, 0);
  const topkv_view_t d = pool_view(TOPKV_LAYOUT_POOL, dst, dst_layer, dst_tables, dst_stride, 0);
  return move_layer(&s, &d, num_reqs, seq_lens, src->num_heads, 0, stream);
}

}  // extern "C"
