// kvcache1.hip - whole-request KV serialization in the KVCACHE1 format and a
// device CRC-64 (declared in include/topkv.h).
//
// Format (paper Section 3.5; field widths, byte order and CRC polynomial are
// this library's reading, documented in topkv.h): a 128-byte header, then
// the K tensor and the V tensor, each [layers][seq_len][kv_heads][head_dim].
// Layer l of a request is written straight into its slices of both tensors
// by the pack kernel with a plane stride of one tensor (topkv_pack_layer_
// planes), so a pipelined sender can ship each layer as soon as it is packed;
// the checksums and header are written once all layers are in.
//
// CRC-64/XZ on the GPU.  Bytes are read LSB-first into a 64-bit register in
// which bit 63 is x^0 ("reflected"); shifting one zero byte in multiplies the
// register by x^8 mod P.  Hence, for the raw register R (preset 0, no final
// complement), R(A || B) = R(A) * x^(8|B|) + R(B) over GF(2), leading zero
// bytes leave R unchanged, and the CRC proper is
// ~(~0 * x^(8N) + R(data)).  Multiplying a register by a fixed power of x is
// linear, so it is the XOR of one lookup per register byte (or nibble) in a
// table of that constant.  Work split:
//   tables: the slicing tables, the constant that advances a register by
//     one sub-chunk and the join levels of the lanes inside a span do not
//     depend on the data; the compiler computes them (kConstTables);
//   kernel 1: the data, front-padded with zero bytes (free, by the property
//     above), is cut into at most 256 equal spans of whole 64 KiB
//     sub-chunks, one 1024-lane workgroup per span (several inputs of one
//     length, such as a blob's K and V tensors, share one launch, each with
//     its share of the spans).  Lane t takes bytes [64t, 64t + 64) of every
//     sub-chunk: a wave loads its 4 KiB slice with fully coalesced 16-byte
//     buffer loads (the next two sub-chunks' in flight while this one is
//     folded; a load in the front padding lies outside the buffer and returns
//     zeros) and hands each lane its 64 bytes through an LDS staging area;
//     lanes run them through slicing-by-4 tables held in LDS in 8 replicas
//     arranged so that the 32 lanes an LDS cycle serves never share a bank
//     (crc_word4), and advance their running register by one sub-chunk per
//     step (a byte-table multiply, its tables in 4 replicas arranged the
//     same way: no LDS lookup of the loop can conflict); a tree of
//     nibble-table multiplies joins
//     the lanes at the end of the span (inside each wave by shuffles, then
//     across the 16 waves), and the span's register is multiplied into its
//     place in the input (one nibble-table multiply per set bit of its
//     distance to the end, in spans).  Nibble sets take twice the lookups of
//     byte sets but an eighth of the room, so they serve where tables are
//     staged or built after the loop, and the byte set where a lookup runs
//     every step;
//   kernel 2: one workgroup XORs each input's placed span registers,
//     appends the sub-16-byte tail, applies the preset and complement, and
//     writes (seal) or checks (verify) a blob's header.
// Shift constants x^(8n) mod P are computed on the host.
//
// One-pass serialization: kernel 1 also runs with the pool as its source
// (kGather: each 16-byte piece of a tensor is loaded from its pool slot
// through the block table, stored to the blob and folded) or its sink
// (kScatter: loaded from the blob, folded and stored to its pool slot), so a
// whole request is serialized or received with the pool and the blob each
// touched once.  A piece's pool slot follows from its tensor offset: the
// sub-chunk's (row, byte) position is carried across sub-chunks as a floor
// quotient and remainder, pieces add their offset with multiply-high
// divisions, and the page entries of the next sub-chunk are loaded while the
// current one is folded.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdint>
#include <cstring>
#include <mutex>

#include "internal.h"
#include "topkv.h"

namespace {

constexpr uint64_t kPolyReflected = 0xC96C5795D7870F42ull;   // ECMA-182, bit-reversed
constexpr int kCrcThreads = 1024;                               // lanes per span workgroup
constexpr int kPiece = 64;                                      // bytes per lane per sub-chunk
constexpr int kLoads = kPiece / 16;                             // 16-byte loads per lane per sub-chunk
constexpr int kSubLog2 = 16;                                    // 64 KiB sub-chunk = 1024 lanes x 64 B
constexpr int64_t kSub = (int64_t)1 << kSubLog2;
constexpr int kMaxSpans = 256;                                  // span workgroups per CRC at most
constexpr int64_t kMaxSpanSubs = 32767;                         // sub-chunks per span at most (span < 2 GiB)
constexpr int kLaneLevels = 10;                                 // log2(kCrcThreads)
constexpr int kSpanLevels = 8;                                  // log2(kMaxSpans)
constexpr int kTableWords = 8 * 256;                            // one set of 8 byte tables (16 KiB)
constexpr int kCopies = 8;                                      // LDS replicas of the slicing tables
constexpr int kSubCopies = 4;                                   // LDS replicas of the advance's tables
constexpr int kWaves = kCrcThreads / 64;
constexpr int kStageWords = kWaves * 64 * 16 / 8;               // per-wave staging of one 1 KiB row
constexpr int kNibWords = 16 * 16;                              // one nibble table set (2 KiB)
// nibble table sets: the lane-join levels
constexpr int kNibSets = kLaneLevels;

struct ShiftConsts {
  uint64_t x8pow2[64];    // x^(8 * 2^k) mod P, reflected
};

__host__ __device__ constexpr uint64_t mul_x(uint64_t w) { return (w >> 1) ^ ((w & 1) ? kPolyReflected : 0); }

// a * b mod P in the reflected representation (bit 63 of a is its x^0 term).
__host__ __device__ constexpr uint64_t mulmod(uint64_t a, uint64_t b) {
  uint64_t prod = 0;
  for (int i = 0; i < 64 && a; ++i) {
    if (a >> 63) prod ^= b;
    a <<= 1;
    b = mul_x(b);
  }
  return prod;
}

const ShiftConsts& shift_consts() {
  static const ShiftConsts c = [] {
    ShiftConsts s;
    uint64_t x8 = 1ull << 63;                                 // x^0
    for (int i = 0; i < 8; ++i) x8 = mul_x(x8);               // x^8
    s.x8pow2[0] = x8;
    for (int k = 1; k < 64; ++k) s.x8pow2[k] = mulmod(s.x8pow2[k - 1], s.x8pow2[k - 1]);
    return s;
  }();
  return c;
}

// x^(8n) mod P from the powers-of-two table (host).
uint64_t x8n(const ShiftConsts& c, uint64_t n) {
  uint64_t r = 1ull << 63;
  for (int k = 0; n; ++k, n >>= 1)
    if (n & 1) r = mulmod(r, c.x8pow2[k]);
  return r;
}

// A set of tables is linear in the register's bits: bit j of a 64-bit value
// stands for the basis word m[j], and an entry is the XOR of m[j] over the
// set bits j of the part of the value it indexes.  Byte sets: entry (k, b) of
// 8 tables covers bits 8k .. 8k + 7; nibble sets: entry (k, n) of 16 tables
// covers bits 4k .. 4k + 3 (16 entries of 8 bytes: one table is 128 bytes, so
// the lanes of an LDS cycle looking up one table never share a bank).
// Slicing set: entry (k, b) is byte b followed by k zero bytes,
// b * x^(8(k + 1)), so m[8k + i] = x^(63 - i) * x^(8k + 8).  Multiply set of
// constant c: entry (k, .) is (value << 8k or 4k) * c, so
// m[j] = x^(63 - j) * c, i.e. m[63] = c and m[j - 1] = x * m[j].  Each entry
// is built from the one with its lowest set bit cleared.
template <int kBits>
__host__ __device__ constexpr void fill_set(uint64_t* set, const uint64_t (&m)[64]) {
  constexpr int kEntries = 1 << kBits;
  for (int k = 0; k < 64 / kBits; ++k) {
    set[k * kEntries] = 0;
    for (int b = 1; b < kEntries; ++b) {
      int low = 0;
      while (!((b >> low) & 1)) ++low;
      set[k * kEntries + b] = set[k * kEntries + (b & (b - 1))] ^ m[kBits * k + low];
    }
  }
}

__host__ __device__ constexpr void multiply_basis(uint64_t (&m)[64], uint64_t c) {
  m[63] = c;
  for (int j = 63; j > 0; --j) m[j - 1] = mul_x(m[j]);
}

// The span-independent table sets, computed by the compiler: the slicing
// bytes, the advance by one sub-chunk (x^(8 * 64 Ki), bytes) and the
// lane-join levels (x^(8 * kPiece * 2^l), nibbles).
struct ConstTables {
  uint64_t slice[kTableWords];
  uint64_t sub[kTableWords];
  uint64_t nib[kNibSets * kNibWords];
};

constexpr ConstTables make_const_tables() {
  ConstTables t{};
  uint64_t p[128] = {};                                      // p[n] = x^n
  p[0] = 1ull << 63;
  for (int n = 1; n < 128; ++n) p[n] = mul_x(p[n - 1]);
  uint64_t m[64] = {};
  for (int k = 0; k < 8; ++k)
    for (int i = 0; i < 8; ++i) m[8 * k + i] = p[71 + 8 * k - i];
  fill_set<8>(t.slice, m);
  uint64_t x8p[kSubLog2 + 1] = {};                           // x8p[k] = x^(8 * 2^k)
  x8p[0] = p[8];
  for (int k = 1; k <= kSubLog2; ++k) x8p[k] = mulmod(x8p[k - 1], x8p[k - 1]);
  multiply_basis(m, x8p[kSubLog2]);
  fill_set<8>(t.sub, m);
  static_assert(kPiece == 64 && 6 + kLaneLevels - 1 <= kSubLog2, "lane levels are x^(8 * 2^(6 + l))");
  for (int l = 0; l < kLaneLevels; ++l) {
    multiply_basis(m, x8p[6 + l]);
    fill_set<4>(t.nib + l * kNibWords, m);
  }
  return t;
}

__device__ const ConstTables kConstTables = make_const_tables();


// Four bytes (little-endian word w) into the register (lo, hi) with
// slicing-by-4 tables (the slicing-by-N method of Kounavis and Berry: one
// table per byte position of the word, the byte's effect after the bytes
// that follow it) held in LDS in kCopies = 8 replicas.  Layout (byte offsets
// in the 64 KiB table region): entry b of table t, replica r sits at
// b * 256 + t * 64 + r * 8, so with the LDS's 64 four-byte banks each (table,
// replica) pair owns banks 16t + 2r and 16t + 2r + 1 whatever the entry.  A
// ds_read_b64 serves 32 lanes at a time; lane l of such a group uses replica
// r = l % 8 and belongs to group g = (l / 8) % 4, and lookup k of group g
// reads table (3 - k + g) % 4: in every instruction the 32 lanes touch 64
// different banks whatever bytes they look up.  Every address is one byte
// permute of the lane's L (byte k: table and replica bytes of lookup k) and
// x = lo ^ w: sel[k] puts L's byte k in byte 0 and the byte of x that table
// looks up in byte 1.  Byte 0 of the word is followed by 3 more bytes (table
// 3), byte 3 by none (table 0).
// a ^ b ^ c in one instruction: gfx950's three-input bitwise operation, truth table 0x96 (bit i of
// the table is the parity of i, the XOR of the three input bits).
__device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t c) {
  return __builtin_amdgcn_bitop3_b32(a, b, c, 0x96);
}

// v times the constant of a nibble set t (16 x 16 words in LDS): one lookup per nibble of v.
__device__ __forceinline__ uint64_t nib_mul(uint64_t v, const uint64_t* t) {
  const uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
  uint2 e[16];
#pragma unroll
  for (int k = 0; k < 16; ++k)
    e[k] = *reinterpret_cast<const uint2*>(t + 16 * k + (((k < 8 ? lo : hi) >> (4 * (k & 7))) & 15));
  uint32_t rl = 0, rh = 0;
#pragma unroll
  for (int k = 0; k < 16; k += 2) {
    rl = xor3(rl, e[k].x, e[k + 1].x);
    rh = xor3(rh, e[k].y, e[k + 1].y);
  }
  return (uint64_t)rh << 32 | rl;
}

// v times the sub-chunk advance: one lookup per byte of v in the advance's byte set, held in LDS in
// kSubCopies = 4 replicas.  Layout (byte offsets in its 64 KiB region): entry b of table t (the table
// of byte t of v), replica r sits at b * 256 + t * 32 + r * 8, so each (table, replica) pair owns one
// pair of the 64 four-byte banks whatever the entry.  Of the 32 lanes an LDS cycle serves, lane l
// uses replica r = l % 4 and belongs to group g = (l / 4) % 8, and lookup k of group g reads table
// (k + g) % 8: in every instruction the 32 lanes sit in 32 different bank pairs.  The lane first
// rotates v right by 8g bits (swap the words when g >= 4, then align by 8 (g % 4)), so lookup k
// always takes byte k of the rotated value; its address is then one byte permute of that word and
// the lane's la / lb (byte k % 4: (32 k + 32 g + 8 r) mod 256, the table and replica bytes).
__device__ __forceinline__ uint64_t sub_advance(uint64_t v, const char* t, uint32_t la, uint32_t lb, bool swap,
                                            uint32_t sh) {
  const uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
  const uint32_t a = swap ? hi : lo, b = swap ? lo : hi;
  const uint32_t w[2] = {__builtin_amdgcn_alignbit(b, a, sh), __builtin_amdgcn_alignbit(a, b, sh)};
  uint2 e[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const uint32_t sel = 0x0c0c0000u | (uint32_t)(k & 3) << 8 | (uint32_t)(4 + (k & 3));
    e[k] = *reinterpret_cast<const uint2*>(t + __builtin_amdgcn_perm(k < 4 ? la : lb, w[k >> 2], sel));
  }
  uint32_t rl = 0, rh = 0;
#pragma unroll
  for (int k = 0; k < 8; k += 2) {
    rl = xor3(rl, e[k].x, e[k + 1].x);
    rh = xor3(rh, e[k].y, e[k + 1].y);
  }
  return (uint64_t)rh << 32 | rl;
}

__device__ __forceinline__ void crc_word4(uint32_t& lo, uint32_t& hi, uint32_t w, const char* tab, uint32_t L,
                                          const uint32_t (&sel)[4]) {
  const uint32_t x = lo ^ w;
  const uint2 e0 = *reinterpret_cast<const uint2*>(tab + __builtin_amdgcn_perm(L, x, sel[0]));
  const uint2 e1 = *reinterpret_cast<const uint2*>(tab + __builtin_amdgcn_perm(L, x, sel[1]));
  const uint2 e2 = *reinterpret_cast<const uint2*>(tab + __builtin_amdgcn_perm(L, x, sel[2]));
  const uint2 e3 = *reinterpret_cast<const uint2*>(tab + __builtin_amdgcn_perm(L, x, sel[3]));
  lo = xor3(xor3(e0.x, e1.x, e2.x), e3.x, hi);
  hi = xor3(e0.y, e1.y, e2.y) ^ e3.y;
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Buffer resource word 3 of an untyped buffer (32-bit data format), and the cache-policy bit of a
// non-temporal buffer access.
constexpr int kBufferWord3 = 0x00020000;
constexpr int kBufferNt = 2;

// n / d for 0 <= n < 2^31 by a multiply-high (Granlund and Montgomery,
// 1994): s = ceil(log2 d), m = floor(2^32 (2^s - d) / d) + 1, and the
// quotient is (mulhi(n, m) + n) >> s.
struct Div32 {
  uint32_t d, m, s;
};

Div32 make_div32(uint32_t d) {
  uint32_t s = 0;
  while ((1ull << s) < d) ++s;
  return Div32{d, (uint32_t)((((1ull << 32) * ((1ull << s) - d)) / d) + 1), s};
}

__device__ __forceinline__ uint32_t div32(uint32_t n, const Div32& f) { return (__umulhi(n, f.m) + n) >> f.s; }

// Where a span kernel's 16-byte pieces come from and go to.  kStream: the
// CRC input is `data`.  kGather: the input is one KVCACHE1 tensor gathered
// from the pool (byte `off` of the tensor is layer first + l, token t, byte b
// of plane `plane_off`'s row), and each piece is also stored to the blob
// tensor; a piece whose page entry is out of range keeps the blob's bytes
// (they are read and folded instead, nothing is written).  kScatter: the
// input is the blob tensor and each piece is also stored to its pool slot
// (pieces of out-of-range pages are not stored).
enum { kStream = 0, kGather = 1, kScatter = 2 };

struct PoolSide {
  char* pool;             // pool base (layer 0)
  u32x4* blob;            // the tensor's first byte in the blob
  const int32_t* table;   // the request's block table
  int64_t layer_bytes, page_bytes, num_pages;
  int64_t plane_off;      // the tensor's plane inside a page row (set per tensor by the kernel)
  int64_t plane_stride;   // between the planes of consecutive tensors
  int64_t step_q;         // kSub / row_bytes
  int32_t step_r;         // kSub mod row_bytes
  int32_t row_bytes, seq_len, page_size, first_layer;
  Div32 d_row, d_seq, d_page;
};

// The factors that place a span's register in its input:
// level[b] = x^(8 * span * 2^b).
struct SpanShift {
  uint64_t level[kSpanLevels];
};

__device__ __forceinline__ uint64_t shfl_xor64(uint64_t v, int mask) {
  const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)v, mask);
  const uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(v >> 32), mask);
  return (uint64_t)hi << 32 | lo;
}

// v of lane + d (lanes past the wave's end keep their own)
__device__ __forceinline__ uint64_t shfl_down64(uint64_t v, int d) {
  const uint32_t lo = (uint32_t)__shfl_down((int)(uint32_t)v, d);
  const uint32_t hi = (uint32_t)__shfl_down((int)(uint32_t)(v >> 32), d);
  return (uint64_t)hi << 32 | lo;
}

// Kernel 1: raw register of each span of the front-padded streams of
// gridDim.x / spans_per_buf inputs (tensors) of `head` bytes each (a multiple
// of 16), input i at data + i * buf_stride bytes (pool modes: the blob tensor
// of plane i); `pad` leading zero bytes (a multiple of 16) make head + pad =
// spans_per_buf spans of span_subs sub-chunks.  Workgroup w takes span
// w % spans_per_buf of input w / spans_per_buf and writes its register,
// multiplied into its place in the input, to
// partial[input * kMaxSpans + span].
template <int kMode>
__global__ __launch_bounds__(kCrcThreads) void crc64_span_kernel(const u32x4* __restrict__ data, int64_t buf_stride,
                                                                 int64_t pad, int64_t span_subs,
                                                                 int32_t spans_per_buf,
                                                                 uint64_t* __restrict__ partial, SpanShift sh,
                                                                 PoolSide ps_in) {
  // One LDS block, laid out by hand so the slicing tables start below 64 KiB (their lookups' table
  // offset then fits the LDS instructions' 16-bit offset field: no address add per lookup):
  // stage_lds: per-wave staging of one 1 KiB row (16 KiB);
  // big: slicing tables 0..3 in kCopies replicas (64 KiB); once every wave has left the loop, the
  // join's tables, the span placement's tables and the waves' registers (layout at the join);
  // sub_lds: the sub-chunk advance's 8 tables in kSubCopies replicas (64 KiB; one OR per lookup).
  __shared__ __attribute__((aligned(16))) uint64_t lds[4 * 256 * kCopies + kTableWords * kSubCopies + kStageWords];
  uint64_t* const stage_lds = lds;
  uint64_t* const big = lds + kStageWords;
  uint64_t* const sub_lds = big + 4 * 256 * kCopies;
  // The table words this thread places in LDS are loaded first; the LDS is filled once the first
  // sub-chunks' loads are also on their way (below), so their latency overlaps the fill.  Thread e
  // places entry e / 4 of slicing table e % 4 and entries (e + 1024 j) / 8 of advance table e % 8
  // (j = 0, 1), so a wave's 32-lane halves write 32 different bank pairs at every step of the fill.
  static_assert(4 * 256 == kCrcThreads, "one slicing entry per thread");
  static_assert(kTableWords == 2 * kCrcThreads, "two sub-chunk advance words per thread");
  const uint32_t fill_t = threadIdx.x & 3, fill_b = threadIdx.x >> 2;
  const uint32_t fill_u = threadIdx.x & 7, fill_c = threadIdx.x >> 3;
  const uint64_t slice_word = kConstTables.slice[fill_t * 256 + fill_b];
  const uint64_t sub_word0 = kConstTables.sub[fill_u * 256 + fill_c];
  const uint64_t sub_word1 = kConstTables.sub[fill_u * 256 + fill_c + kCrcThreads / 8];
  __builtin_amdgcn_sched_barrier(0);
  // this workgroup's input and span
  const int32_t buf_idx = (int32_t)blockIdx.x / spans_per_buf;
  const int32_t span_idx = (int32_t)blockIdx.x - buf_idx * spans_per_buf;
  PoolSide ps = ps_in;
  ps.plane_off = buf_idx * ps_in.plane_stride;
  if (kMode != kStream) ps.blob += buf_idx * (buf_stride / 16);
  data += buf_idx * (buf_stride / 16);
  const char* tab = reinterpret_cast<const char*>(big);
  // this lane's table-and-replica bytes and the permute selectors of crc_word4's four lookups:
  // lookup k reads table t = (3 - k + g) % 4 (selector bytes: 4 + k -> L.b(k), 3 - t -> x.b(3 - t),
  // 0x0c -> zero)
  static_assert(kCopies == 8, "8 replicas x 4 groups = the 32 lanes of an LDS cycle");
  const uint32_t rep8 = threadIdx.x & 7, grp4 = (threadIdx.x >> 3) & 3;
  uint32_t L = 0;
  uint32_t sel[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const uint32_t t = (3u - (uint32_t)k + grp4) & 3u;
    L |= (t * 64u + rep8 * 8u) << (8 * k);
    sel[k] = 0x0c0c0000u | (3u - t) << 8 | (4u + (uint32_t)k);
  }
  // the advance's lane constants (layout at sub_advance): replica l % 4, group (l / 4) % 8
  static_assert(kSubCopies == 4, "4 replicas x 8 groups = the 32 lanes of an LDS cycle");
  const uint32_t rep4 = threadIdx.x & 3, grp8 = (threadIdx.x >> 2) & 7;
  const bool adv_swap = grp8 >= 4;
  const uint32_t adv_sh = 8u * (grp8 & 3u);
  uint32_t adv_la = 0, adv_lb = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    adv_la |= ((32u * (uint32_t)k + 32u * grp8 + 8u * rep4) & 255u) << (8 * k);
    adv_lb |= ((32u * (uint32_t)(k + 4) + 32u * grp8 + 8u * rep4) & 255u) << (8 * k);
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // this wave's 1 KiB staging area: one row of 64 16-byte slots, used once per row of the wave's
  // 4 KiB of a sub-chunk; slot l holds the row's bytes [16 l, +16) at position l ^ ((l >> 4) & 3),
  // which keeps both the row writes and the lane-piece reads free of bank conflicts
  u32x4* stage_area = reinterpret_cast<u32x4*>(stage_lds) + wave * 64;
  const char* t_sub = reinterpret_cast<const char*>(sub_lds);      // the sub-chunk advance (LDS)
  // this lane's 16-byte column within a sub-chunk, and the first sub-chunk's data offset
  const int32_t local = wave * 64 * kPiece + 16 * lane;
  const int64_t span0 = (int64_t)span_idx * span_subs * kSub - pad;
  const int64_t base = span0 + local;

  // Pool side.  A sub-chunk's first tensor byte sb is tracked as the floor
  // quotient and remainder (r0, in0) of sb / row_bytes (sb < 0 in the front
  // padding gives r0 < 0): one step of kSub bytes adds (step_q, step_r) with a
  // carry.  A piece at x = in0 + its offset inside the sub-chunk then lies in
  // row r0 + x / row_bytes (rows < 0: padding) at byte x mod row_bytes.
  struct RowPos {
    int64_t r0;
    int32_t in0;
  };
  auto advance = [&](RowPos p) {
    p.in0 += ps.step_r;
    p.r0 += ps.step_q;
    if (p.in0 >= ps.row_bytes) {
      p.in0 -= ps.row_bytes;
      ++p.r0;
    }
    return p;
  };
  RowPos pos0;
  if (kMode != kStream) {
    const int64_t q = span0 >= 0 ? span0 / ps.row_bytes : -((-span0 + ps.row_bytes - 1) / ps.row_bytes);
    pos0 = RowPos{q, (int32_t)(span0 - q * ps.row_bytes)};
  }
  // the piece's (layer-major) row and its byte in the row; false in the padding
  auto row_of = [&](const RowPos& p, int j, uint32_t* row, uint32_t* inrow) -> bool {
    const uint32_t x = (uint32_t)(p.in0 + local + 1024 * j);
    const uint32_t q = div32(x, ps.d_row);
    const int64_t r = p.r0 + q;
    if (r < 0) return false;
    *row = (uint32_t)r;
    *inrow = x - q * (uint32_t)ps.row_bytes;
    return true;
  };
  // A piece's pool offset splits into a page-independent part pb (layer,
  // plane, slot and byte; -1 in the padding), worked out once per piece
  // together with its table index, and the page entry pg loaded from the
  // table: offset = pb + pg * page_bytes (one 32 x 32 -> 64-bit multiply-add).
  // (Every piece loads an entry - a padding piece row 0's - and the padding is marked in pb alone, so
  // no branch surrounds a load and nothing waits for the entries until a piece's slot is needed.)
  auto piece = [&](const RowPos& p, int j, uint32_t* idx) -> int64_t {
    uint32_t row = 0, inrow = 0;
    const bool in_tensor = row_of(p, j, &row, &inrow);
    const uint32_t l = div32(row, ps.d_seq);
    const uint32_t t = row - l * (uint32_t)ps.seq_len;
    const uint32_t i = div32(t, ps.d_page);                      // < ceil(seq_len / page_size)
    *idx = i;
    return in_tensor ? (int64_t)(ps.first_layer + (int32_t)l) * ps.layer_bytes + ps.plane_off +
                           (int64_t)((uint64_t)(t - i * (uint32_t)ps.page_size) * (uint32_t)ps.row_bytes) + inrow
                     : -1;
  };
  auto lookup = [&](int64_t (&pb)[kLoads], int32_t (&pg)[kLoads], const RowPos& p) {
#pragma unroll
    for (int j = 0; j < kLoads; ++j) {
      uint32_t i = 0;
      pb[j] = piece(p, j, &i);
      pg[j] = ps.table[i];
    }
  };
  // (kScatter) the entries alone, loaded a step ahead, and the page-independent offsets worked out
  // again where the pieces are stored: fewer registers carried from step to step
  auto entries = [&](int32_t (&pg)[kLoads], const RowPos& p) {
#pragma unroll
    for (int j = 0; j < kLoads; ++j) {
      uint32_t i = 0;
      (void)piece(p, j, &i);
      pg[j] = ps.table[i];
    }
  };
  auto offsets = [&](int64_t (&pb)[kLoads], const RowPos& p) {
#pragma unroll
    for (int j = 0; j < kLoads; ++j) {
      uint32_t i = 0;
      pb[j] = piece(p, j, &i);
    }
  };
  // pool byte of a piece: -1 in the padding, -2 when its page entry is out of range
  auto slot_of = [&](int64_t pb, int32_t page) -> int64_t {
    if (pb < 0) return -1;
    if (page < 0 || (int64_t)page >= ps.num_pages) return -2;
    return pb + (int64_t)((uint64_t)(uint32_t)page * (uint32_t)ps.page_bytes);
  };
  const u32x4 zero = {0u, 0u, 0u, 0u};
  const u32x4* in = kMode == kScatter ? ps.blob : data;

  // kStream / kScatter: contiguous input (the data, or the blob tensor)
  // Every load is issued (the front padding's at offset 0: no branch around a load, so the compiler
  // counts outstanding loads exactly); bit j of *pad marks a piece of the padding, which the staging
  // step replaces by zeros when the data is used.
  // Buffer loads relative to the workgroup's first input byte, with a 32-bit lane offset (spans are
  // shorter than 2 GiB).  In the front padding the offset is negative, i.e. above the resource's
  // size as an unsigned number, and such a load returns zeros without touching memory: the padding's
  // zero bytes come from the load itself.
  const int64_t in_lo = span0 > 0 ? span0 : 0;
  const __amdgpu_buffer_rsrc_t in_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<char*>(reinterpret_cast<const char*>(in)) + in_lo, (short)0,
      (int)(span0 + span_subs * kSub - in_lo), kBufferWord3);
  const int32_t lane_off = local + (int32_t)(span0 - in_lo);
  auto load = [&](u32x4 (&v)[kLoads], int64_t sub, uint32_t* pad) {
    *pad = 0;
#pragma unroll
    for (int j = 0; j < kLoads; ++j) {
      const int32_t off = lane_off + ((int32_t)sub << kSubLog2) + 1024 * j;
      v[j] = __builtin_amdgcn_raw_buffer_load_b128(in_rsrc, (uint32_t)off, 0, kBufferNt);
    }
  };
  // kGather: pool pieces (page entries pg loaded an iteration earlier); bad pages read the blob.
  // Bit j of *moved: piece j came from the pool (so the blob store writes it).
  auto gather = [&](u32x4 (&v)[kLoads], int64_t sub, const int64_t (&pb)[kLoads], const int32_t (&pg)[kLoads],
                    uint32_t* moved, uint32_t* pad) {
    *moved = 0;
    *pad = 0;
#pragma unroll
    for (int j = 0; j < kLoads; ++j) {
      const int64_t po = slot_of(pb[j], pg[j]);
      const int64_t off = base + (sub << kSubLog2) + 1024 * j;
      // one load per piece whatever its source (the padding's from the blob's start)
      const u32x4* src = po >= 0 ? reinterpret_cast<const u32x4*>(ps.pool + po) : ps.blob + (po == -2 ? off / 16 : 0);
      v[j] = __builtin_nontemporal_load(src);
      *moved |= (po >= 0 ? 1u : 0u) << j;
      *pad |= (po == -1 ? 1u : 0u) << j;
    }
  };
  auto put_blob = [&](const u32x4 (&v)[kLoads], int64_t sub, uint32_t moved) {
#pragma unroll
    for (int j = 0; j < kLoads; ++j)
      if (moved >> j & 1) __builtin_nontemporal_store(v[j], ps.blob + (base + (sub << kSubLog2) + 1024 * j) / 16);
  };
  auto put_pool = [&](const u32x4 (&v)[kLoads], const int64_t (&pb)[kLoads], const int32_t (&pg)[kLoads]) {
#pragma unroll
    for (int j = 0; j < kLoads; ++j) {
      const int64_t po = slot_of(pb[j], pg[j]);
      if (po >= 0) __builtin_nontemporal_store(v[j], reinterpret_cast<u32x4*>(ps.pool + po));
    }
  };
  const int wr = lane ^ ((lane >> 4) & 3);                        // write slot of this lane in each row
  const int rrow = lane >> 4, rcol = 4 * (lane & 15);             // this lane's piece: row, first column
  uint64_t fold = 0;
  // Per-sub-chunk state in kDepth sets used in turn, so a step never copies a later sub-chunk's
  // registers (a copy would wait for its loads): the pieces, the padding and moved masks, and (pool
  // modes) the page entries and (kGather) the page-independent offsets.  The streaming mode keeps two sub-chunks'
  // loads in flight while it folds a third; the pool modes, which need more registers per piece, one.
  constexpr int kDepth = kMode == kStream ? 3 : 2;
  u32x4 buf[kDepth][kLoads];
  int64_t pb[kDepth][kLoads] = {};
  int32_t pg[kDepth][kLoads] = {};
  uint32_t zp[kDepth] = {}, mv[kDepth] = {};
  RowPos pos = pos0;   // row position of the sub-chunk the next step folds (pool modes)
  if (kMode == kGather) {
    lookup(pb[0], pg[0], pos);
    gather(buf[0], 0, pb[0], pg[0], &mv[0], &zp[0]);
    if (span_subs > 1) lookup(pb[1], pg[1], advance(pos));
  } else {
    // in set order, as the loop issues them (kept apart so the scheduler cannot interleave the sets:
    // the loop's waits count loads in issue order, and a set issued later than the loop assumes would
    // make every iteration wait for it)
#pragma unroll
    for (int k = 0; k + 1 < kDepth; ++k) {
      load(buf[k], k < span_subs ? k : span_subs - 1, &zp[k]);
      __builtin_amdgcn_sched_barrier(0);
    }
    if (kMode == kScatter) entries(pg[0], pos);
  }
  {
    // every replica of this thread's entries (layouts at crc_word4 and sub_advance), replica
    // (i + lane / 4) % 8 resp. (i + lane / 8) % 4 at step i
    char* srow = reinterpret_cast<char*>(big) + fill_b * 256 + fill_t * 64;
#pragma unroll
    for (int i = 0; i < kCopies; ++i)
      *reinterpret_cast<uint64_t*>(srow + ((i + (threadIdx.x >> 2)) & (kCopies - 1)) * 8) = slice_word;
    char* arow = reinterpret_cast<char*>(sub_lds) + fill_c * 256 + fill_u * 32;
#pragma unroll
    for (int i = 0; i < kSubCopies; ++i) {
      const int r = (i + (threadIdx.x >> 3)) & (kSubCopies - 1);
      *reinterpret_cast<uint64_t*>(arow + r * 8) = sub_word0;
      *reinterpret_cast<uint64_t*>(arow + (kCrcThreads / 8) * 256 + r * 8) = sub_word1;
    }
  }
  __syncthreads();
  // One step: fold sub-chunk `sub` (set c) while the loads of sub-chunk sub + kDepth - 1 go into set n
  // (the set the previous step folded).  Every step of a loop iteration runs, also past the span's
  // end: such a step's loads reread the span's last sub-chunk (so no branch surrounds a load and the
  // compiler's count of outstanding loads is exact on every path) and the rest of it is skipped.
  auto step = [&](int64_t sub, int c, int n) {
    const bool live = sub < span_subs;
    const int64_t ahead = sub + kDepth - 1;
    if (kMode == kGather) {
      // entries of sub + 1 were looked up a step ago into set n; set c's entries are free once sub's
      // pieces are in, and take those of sub + 2
      if (live) {
        const RowPos p1 = advance(pos);
        if (sub + 1 < span_subs) gather(buf[n], sub + 1, pb[n], pg[n], &mv[n], &zp[n]);
        put_blob(buf[c], sub, mv[c]);
        if (sub + 2 < span_subs) lookup(pb[c], pg[c], advance(p1));
        pos = p1;
      }
    } else {
      load(buf[n], ahead < span_subs ? ahead : span_subs - 1, &zp[n]);
      if (kMode == kScatter && live) {
        // the next sub-chunk's entries (on a span's last step past the tensor's end: in-range table
        // indices whose entries are never used), then this sub-chunk's pieces to their pool slots
        const RowPos p1 = advance(pos);
        entries(pg[n], p1);
        int64_t pbc[kLoads];
        offsets(pbc, pos);
        put_pool(buf[c], pbc, pg[c]);
        pos = p1;
      }
    }
    if (!live) return;
    // the advance of the running register by one sub-chunk (LDS lookups; they return while this
    // sub-chunk's bytes are folded; the sender, shortest of registers, takes it after the fold)
    uint64_t adv = 0;
    if (kMode != kGather) adv = sub_advance(fold, t_sub, adv_la, adv_lb, adv_swap, adv_sh);
    u32x4 piece[kLoads];
    // (kGather) pieces of the front padding, only in a sub-chunk that starts before the data (the same
    // for the whole workgroup), are staged as zeros
    const bool front = kMode == kGather && span0 + (sub << kSubLog2) < 0;
#pragma unroll
    for (int h = 0; h < kLoads; ++h) {   // row h: lanes 16h .. 16h + 15 take their pieces
      if (front)
        stage_area[wr] = (zp[c] >> h & 1) ? zero : buf[c][h];
      else
        stage_area[wr] = buf[c][h];
      __builtin_amdgcn_wave_barrier();
      if (rrow == h) {
#pragma unroll
        for (int m = 0; m < kLoads; ++m) {
          const int l = rcol + m;
          piece[m] = stage_area[l ^ ((l >> 4) & 3)];
        }
      }
      __builtin_amdgcn_wave_barrier();   // reads done before the next writes
    }
    uint32_t lo = 0, hi = 0;
#pragma unroll
    for (int j = 0; j < kLoads; ++j) {
      crc_word4(lo, hi, piece[j].x, tab, L, sel);
      crc_word4(lo, hi, piece[j].y, tab, L, sel);
      crc_word4(lo, hi, piece[j].z, tab, L, sel);
      crc_word4(lo, hi, piece[j].w, tab, L, sel);
    }
    if (kMode == kGather) adv = sub_advance(fold, t_sub, adv_la, adv_lb, adv_swap, adv_sh);
    fold = adv ^ ((uint64_t)hi << 32 | lo);
  };
  for (int64_t sub = 0; sub < span_subs; sub += kDepth) {
#pragma unroll
    for (int k = 0; k < kDepth; ++k) step(sub + k, k, (k + kDepth - 1) % kDepth);
  }
  // Join the lanes: lanes t and t + s (the later s lanes x kPiece bytes of every sub-chunk) give t's
  // register times x^(8 * kPiece * s) plus t + s's register, s = 1, 2, ..., 512 lanes: levels 0..5
  // inside each wave by shuffles, levels 6..9 across the 16 waves, with the levels' nibble sets.
  // Then the span's register times X^k, X = x^(8 * span), k = spans_per_buf - 1 - span_idx: its place
  // in the input, so that the registers of an input's spans just XOR together.  One factor
  // x^(8 * span * 2^b) per set bit b of k; wave b works out the basis of factor b (lane p holds
  // x^(63 - p) times it) and turns it into the factor's nibble set.  The join's sets and the bases are
  // loaded and worked out as each wave leaves the loop, while others may still be folding.
  static_assert(kNibSets * kNibWords <= 3 * kCrcThreads, "three join words per thread");
  uint64_t jw[3];
#pragma unroll
  for (int j = 0; j < 3; ++j) {
    const int e = j * kCrcThreads + threadIdx.x;
    jw[j] = e < kNibSets * kNibWords ? kConstTables.nib[e] : 0ull;
  }
  const int k = spans_per_buf - 1 - span_idx;
  const bool place = wave < kSpanLevels && ((k >> wave) & 1);
  uint64_t bw = 0;
  if (place) {
    bw = sh.level[wave];
    for (int it = 0; it < 63; ++it)
      if (it < 63 - lane) bw = mul_x(bw);
  }
  __syncthreads();   // every lane is done with the slicing tables and the staging area
  // big (words): [0, 2560) the join's nibble sets, [3072, 5120) the placement factors' nibble sets,
  // [5120, 5632) their bases, [5632, 5648) the waves' registers
  uint64_t* lane_nib = big;
  uint64_t* place_nib = big + 3072;
  uint64_t* basis = big + 5120;
  uint64_t* wave_reg = big + 5632;
  static_assert(kNibSets * kNibWords <= 3072 && 3072 + kSpanLevels * kNibWords <= 5120 &&
                    5120 + kSpanLevels * 64 <= 5632 && 5632 + kWaves <= 4 * 256 * kCopies,
                "join and placement layout fits the table region");
#pragma unroll
  for (int j = 0; j < 3; ++j) {
    const int e = j * kCrcThreads + threadIdx.x;
    if (e < kNibSets * kNibWords) lane_nib[e] = jw[j];
  }
  if (place) basis[wave * 64 + lane] = bw;
  __syncthreads();
  uint64_t acc = fold;
#pragma unroll
  for (int l = 0; l < 6; ++l) {
    const uint64_t later = shfl_down64(acc, 1 << l);
    acc = nib_mul(acc, lane_nib + l * kNibWords) ^ later;
  }
  if (lane == 0) wave_reg[wave] = acc;
  if (place) {
    // entries 4 lane .. 4 lane + 3 of factor `wave`'s nibble set: entry (q, n), q = lane / 4,
    // n = 4 (lane % 4) + j, is the XOR of basis words 4q + i over the set bits i of n
    const uint64_t* m = basis + wave * 64 + 4 * (lane >> 2);
    const uint64_t m0 = m[0], m1 = m[1], m2 = m[2], m3 = m[3];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = 4 * (lane & 3) + j;
      place_nib[wave * kNibWords + 4 * lane + j] =
          ((n & 1) ? m0 : 0ull) ^ ((n & 2) ? m1 : 0ull) ^ ((n & 4) ? m2 : 0ull) ^ ((n & 8) ? m3 : 0ull);
    }
  }
  __syncthreads();
  if (wave == 0) {
    // lanes 0..15 hold the waves' registers (wave w: bytes [4 KiB w, 4 KiB (w + 1)) of every sub-chunk)
    uint64_t a = wave_reg[lane & (kWaves - 1)];
#pragma unroll
    for (int l = 6; l < kLaneLevels; ++l) {
      const uint64_t later = shfl_down64(a, 1 << (l - 6));
      a = nib_mul(a, lane_nib + l * kNibWords) ^ later;
    }
    uint64_t r = a;
    for (int bit = 0; bit < kSpanLevels; ++bit)
      if ((k >> bit) & 1) r = nib_mul(r, place_nib + bit * kNibWords);
    if (lane == 0) partial[buf_idx * kMaxSpans + span_idx] = r;
  }
}

// The KVCACHE1 header (written by seal, checked by verify): sixteen
// little-endian 8-byte words, words 8 and 9 the checksums of K and V.
struct HeaderFields {
  uint64_t request_id, model_id;
  uint32_t seq_len, layers, kv_heads, head_dim, elem_bytes, planes;
  uint64_t k_bytes, v_bytes;
};

__device__ uint64_t header_word(const HeaderFields& f, int w, const uint64_t* crcs) {
  switch (w) {
    case 0: {
      uint64_t magic;
      memcpy(&magic, "KVCACHE1", 8);
      return magic;
    }
    case 1: return f.request_id;
    case 2: return f.model_id;
    case 3: return (uint64_t)f.seq_len | ((uint64_t)f.layers << 32);
    case 4: return (uint64_t)f.kv_heads | ((uint64_t)f.head_dim << 32);
    case 5: return (uint64_t)f.elem_bytes | ((uint64_t)f.planes << 32);
    case 6: return f.k_bytes;
    case 7: return f.v_bytes;
    case 8: return crcs[0];
    case 9: return crcs[1];
    default: return 0;
  }
}

// What kernel 2 does with the checksums: write them out, also write a blob's
// header with them (seal), or also check a blob's header against them
// (verify: result[0] = TOPKV_OK or TOPKV_ERR_CHECKSUM, result[1] = mask of
// bad header words 0..7, result[2] / [3] = K / V checksum mismatch).
enum { kFinishCrcs = 0, kFinishSeal = 1, kFinishVerify = 2 };

struct FinishArgs {
  int32_t inputs;                       // inputs with data (span registers and tails)
  int32_t outputs;                      // checksums produced (inputs, then empty ones: CRC 0)
  int32_t spans, tail_len;
  int64_t stride;                       // between the inputs' tails
  uint64_t preset_shift;                // ~0 * x^(8n): the preset carried over the n bytes
  int32_t what;
  HeaderFields f;
};

// Kernel 2 (one workgroup of kMaxSpans lanes): each input's span registers,
// already in place, XOR into its raw register R; the tail bytes are appended
// and the CRC finished, out[i] = ~(preset_shift + R); then the header is
// written or checked.
__global__ __launch_bounds__(kMaxSpans) void crc64_finish_kernel(const uint64_t* __restrict__ partial,
                                                                 const unsigned char* __restrict__ tail,
                                                                 FinishArgs a, uint64_t* __restrict__ out,
                                                                 unsigned char* __restrict__ blob,
                                                                 int32_t* __restrict__ result) {
  __shared__ uint64_t t0[256];
  __shared__ uint64_t part[2][kMaxSpans / 64];
  __shared__ uint64_t crcs[2];
  static_assert(kMaxSpans == 256, "one slicing-table entry per lane");
  const int i = threadIdx.x, lane = i & 63, wave = i >> 6;
  t0[i] = kConstTables.slice[i];                                  // slicing table 0
  for (int in = 0; in < a.inputs; ++in) {
    uint64_t v = i < a.spans ? partial[in * kMaxSpans + i] : 0ull;
    for (int o = 32; o > 0; o >>= 1) v ^= shfl_xor64(v, o);
    if (lane == 0) part[in][wave] = v;
  }
  __syncthreads();
  if (i < a.outputs) {
    uint64_t c = 0;                                             // the CRC of no bytes
    if (i < a.inputs) {
      uint64_t r = part[i][0] ^ part[i][1] ^ part[i][2] ^ part[i][3];
      const unsigned char* tl = tail + i * a.stride;
      for (int b = 0; b < a.tail_len; ++b) r = t0[(r ^ tl[b]) & 0xff] ^ (r >> 8);
      c = ~(a.preset_shift ^ r);
    }
    out[i] = c;
    crcs[i] = c;
  }
  if (a.what == kFinishCrcs) return;
  __syncthreads();
  if (a.what == kFinishSeal) {
    if (i < 16) reinterpret_cast<uint64_t*>(blob)[i] = header_word(a.f, i, crcs);
  } else if (i == 0) {
    const uint64_t* h = reinterpret_cast<const uint64_t*>(blob);
    int32_t bad = 0;
    for (int w = 0; w < 8; ++w)
      if (h[w] != header_word(a.f, w, crcs)) bad |= 1 << w;
    const int32_t ck = h[8] != crcs[0];
    const int32_t cv = h[9] != crcs[1];
    result[0] = (bad | ck | cv) ? (int32_t)TOPKV_ERR_CHECKSUM : (int32_t)TOPKV_OK;
    result[1] = bad;
    result[2] = ck;
    result[3] = cv;
  }
}

// Workspace words one CRC needs: its span registers.
int64_t crc_words(int64_t) { return kMaxSpans; }

// Span geometry of CRCs over `inputs` inputs of n bytes each, launched
// together: each 16-byte-aligned head is cut into `spans` spans of
// `span_subs` sub-chunks (spans <= kMaxSpans / inputs, so all inputs' spans
// fill one launch of at most kMaxSpans workgroups).
struct Spans {
  int64_t head, span_subs, span, spans;
};

Spans span_geometry(int64_t n, int inputs = 1) {
  Spans g;
  const int64_t max_spans = kMaxSpans / inputs;
  g.head = n - n % 16;
  const int64_t subs = (g.head + kSub - 1) / kSub;
  g.span_subs = subs > 0 ? (subs + max_spans - 1) / max_spans : 1;
  g.span = g.span_subs * kSub;
  g.spans = (g.head + g.span - 1) / g.span;
  return g;
}

// Kernel 2's arguments for CRCs of `inputs` inputs of n bytes, `stride` apart,
// whose spans follow span_geometry(n, inputs): checksums only.
FinishArgs finish_args(int64_t n, int inputs, int64_t stride) {
  const ShiftConsts& sc = shift_consts();
  const Spans g = span_geometry(n, inputs);
  FinishArgs a{};
  a.inputs = inputs;
  a.outputs = inputs;
  a.spans = (int32_t)g.spans;
  a.tail_len = (int32_t)(n - g.head);
  a.stride = stride;
  a.preset_shift = mulmod(x8n(sc, (uint64_t)n), ~0ull);
  a.what = kFinishCrcs;
  return a;
}

SpanShift span_shift(int64_t span) {
  SpanShift s;
  s.level[0] = x8n(shift_consts(), (uint64_t)span);
  for (int b = 1; b < kSpanLevels; ++b) s.level[b] = mulmod(s.level[b - 1], s.level[b - 1]);
  return s;
}

// Queue the CRC-64/XZ of each of a.inputs inputs of n bytes, input i at
// data + i * a.stride (16-byte aligned), into out[0 .. a.outputs) (device),
// then what a.what asks for (blob: the header; result: verify's four words).
// partial has room for a.inputs * kMaxSpans words.
topkv_status_t crc64_launch(const unsigned char* data, int64_t n, const FinishArgs& a, uint64_t* partial,
                            uint64_t* out, unsigned char* blob, int32_t* result, hipStream_t stream) {
  const Spans g = span_geometry(n, a.inputs);
  if (g.span_subs > kMaxSpanSubs) return TOPKV_ERR_UNSUPPORTED;   // spans of 2 GiB and more
  if (g.spans > 0) {
    hipLaunchKernelGGL(crc64_span_kernel<kStream>, dim3((unsigned)(g.spans * a.inputs)), dim3(kCrcThreads), 0,
                       stream, reinterpret_cast<const u32x4*>(data), a.stride, g.spans * g.span - g.head,
                       g.span_subs, (int32_t)g.spans, partial, span_shift(g.span), PoolSide{});
    if (hipGetLastError() != hipSuccess) return TOPKV_ERR_LAUNCH;
  }
  hipLaunchKernelGGL(crc64_finish_kernel, dim3(1), dim3(kMaxSpans), 0, stream, partial, data + g.head, a, out, blob,
                     result);
  return hipGetLastError() == hipSuccess ? TOPKV_OK : TOPKV_ERR_LAUNCH;
}

// ---------------------------------------------------------------------------
// KVCACHE1
// ---------------------------------------------------------------------------

constexpr int64_t kHeaderBytes = 128;

struct Blob {
  int64_t row, k_bytes, v_bytes, total;
};

topkv_status_t blob_geometry(const topkv_pool_t* g, int32_t seq_len, Blob* b) {
  if (!g || seq_len < 0 || g->num_layers <= 0 || g->planes <= 0 || g->planes > 2 || g->num_heads <= 0 ||
      g->head_dim <= 0 || g->elem_bytes <= 0)
    return TOPKV_ERR_INVALID_ARG;
  int64_t row, tensor;
  if (__builtin_mul_overflow((int64_t)g->num_heads * g->head_dim, (int64_t)g->elem_bytes, &row) ||
      __builtin_mul_overflow(row, (int64_t)seq_len, &tensor) ||
      __builtin_mul_overflow(tensor, (int64_t)g->num_layers, &tensor) || tensor > INT64_MAX / 2 - kHeaderBytes)
    return TOPKV_ERR_UNSUPPORTED;
  if (row % 16) return TOPKV_ERR_UNSUPPORTED;   // tensors must stay 16-byte aligned inside the blob
  b->row = row;
  b->k_bytes = tensor;
  b->v_bytes = g->planes == 2 ? tensor : 0;
  b->total = kHeaderBytes + b->k_bytes + b->v_bytes;
  return TOPKV_OK;
}

HeaderFields fields(const topkv_pool_t* g, int32_t seq_len, uint64_t request_id, uint64_t model_id, const Blob& b) {
  HeaderFields f;
  f.request_id = request_id;
  f.model_id = model_id;
  f.seq_len = (uint32_t)seq_len;
  f.layers = (uint32_t)g->num_layers;
  f.kv_heads = (uint32_t)g->num_heads;
  f.head_dim = (uint32_t)g->head_dim;
  f.elem_bytes = (uint32_t)g->elem_bytes;
  f.planes = (uint32_t)g->planes;
  f.k_bytes = (uint64_t)b.k_bytes;
  f.v_bytes = (uint64_t)b.v_bytes;
  return f;
}

// Both checksums of a blob body into ws[0..1] (then the span registers), and
// the header written (kFinishSeal) or checked (kFinishVerify, into result).
topkv_status_t blob_crcs(unsigned char* blob, const Blob& b, const HeaderFields& f, int what, int32_t* result,
                         uint64_t* ws, hipStream_t stream) {
  const int inputs = b.v_bytes == b.k_bytes ? 2 : 1;   // an MLA blob has no V tensor
  FinishArgs a = finish_args(b.k_bytes, inputs, b.k_bytes);
  a.outputs = 2;
  a.what = what;
  a.f = f;
  return crc64_launch(blob + kHeaderBytes, b.k_bytes, a, ws + 2, ws, blob, result, stream);
}

int64_t blob_ws_bytes(const Blob& b) {
  return (int64_t)sizeof(uint64_t) * (2 + 2 * kMaxSpans);
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

// Whether the span kernels can move a whole request's tensors between the pool
// and the blob themselves (32-bit row and token arithmetic, 16-byte pieces).
bool fused_fits(const topkv_pool_t* pool, int32_t seq_len, const Blob& b) {
  return seq_len > 0 && (int64_t)pool->num_layers * seq_len < INT32_MAX && b.row < INT32_MAX - 2 * kSub &&
         (int64_t)pool->planes * pool->page_size * b.row <= UINT32_MAX && aligned16(pool->base) &&
         span_geometry(b.k_bytes, pool->planes).span_subs <= kMaxSpanSubs;
}

// Both checksums of the blob body into ws[0..1] while the K and V tensors of
// every layer move between the pool and the blob inside the span kernels
// (kGather: pool -> blob, kScatter: blob -> pool).
template <int kMode>
topkv_status_t fused_blob_crcs(const topkv_pool_t* pool, const int32_t* table, int32_t seq_len, unsigned char* blob,
                               const Blob& b, const HeaderFields& f, int what, int32_t* result, uint64_t* ws,
                               hipStream_t stream) {
  PoolSide ps{};
  ps.pool = static_cast<char*>(pool->base);
  ps.table = table;
  ps.row_bytes = (int32_t)b.row;
  ps.page_size = pool->page_size;
  ps.page_bytes = (int64_t)pool->planes * pool->page_size * b.row;
  ps.layer_bytes = pool->num_pages * ps.page_bytes;
  ps.num_pages = pool->num_pages;
  ps.seq_len = seq_len;
  ps.first_layer = 0;
  ps.step_q = kSub / b.row;
  ps.step_r = (int32_t)(kSub % b.row);
  ps.d_row = make_div32((uint32_t)b.row);
  ps.d_seq = make_div32((uint32_t)seq_len);
  ps.d_page = make_div32((uint32_t)pool->page_size);
  // every plane's tensor (K, V) in one launch of each kernel; the tensors have the same size (tensors
  // are whole 16-byte rows: no tail); an MLA cache has no V tensor: its checksum is that of no bytes
  const Spans g = span_geometry(b.k_bytes, pool->planes);
  FinishArgs a = finish_args(b.k_bytes, pool->planes, b.k_bytes);
  a.outputs = 2;
  a.what = what;
  a.f = f;
  ps.plane_stride = (int64_t)pool->page_size * b.row;
  ps.blob = reinterpret_cast<u32x4*>(blob + kHeaderBytes);
  hipLaunchKernelGGL(crc64_span_kernel<kMode>, dim3((unsigned)(g.spans * pool->planes)), dim3(kCrcThreads), 0, stream,
                     ps.blob, b.k_bytes, g.spans * g.span - g.head, g.span_subs, (int32_t)g.spans, ws + 2,
                     span_shift(g.span), ps);
  if (hipGetLastError() != hipSuccess) return TOPKV_ERR_LAUNCH;
  hipLaunchKernelGGL(crc64_finish_kernel, dim3(1), dim3(kMaxSpans), 0, stream, ws + 2,
                     reinterpret_cast<const unsigned char*>(ps.blob) + g.head, a, ws, blob, result);
  return hipGetLastError() == hipSuccess ? TOPKV_OK : TOPKV_ERR_LAUNCH;
}

// Layers [first_layer, first_layer + num_layers) of one request into (pack) or
// out of (unpack) their rows of the blob's K and V tensors: grids of
// topkv_engine_layers_per_grid layers when the layer dimension fits the
// direct grid, else one launch per layer.
topkv_status_t kv1_move_layers(bool pack, const topkv_pool_t* pool, int32_t first_layer, int32_t num_layers,
                                      const int32_t* block_table, int32_t seq_len, void* blob, int64_t blob_bytes,
                                      hipStream_t stream) {
  Blob b;
  topkv_status_t st = blob_geometry(pool, seq_len, &b);
  if (st != TOPKV_OK) return st;
  if (!blob || blob_bytes < b.total || first_layer < 0 || num_layers < 0 ||
      (int64_t)first_layer + num_layers > pool->num_layers)
    return TOPKV_ERR_INVALID_ARG;
  if (!aligned16(blob)) return TOPKV_ERR_UNSUPPORTED;
  if (seq_len == 0 || num_layers == 0) return TOPKV_OK;
  const int64_t layer_rows = (int64_t)seq_len * b.row;                 // one layer's rows in one tensor
  unsigned char* k = static_cast<unsigned char*>(blob) + kHeaderBytes + first_layer * layer_rows;
  const int64_t cap = blob_bytes - (kHeaderBytes + first_layer * layer_rows);
  // grids of the layer engine's length (the same measured effect: one grid over a long range of
  // layers moves them slower than a few shorter grids back to back)
  const int32_t per = topkv_engine_layers_per_grid(num_layers, (int64_t)pool->planes * layer_rows, nullptr);
  if (per < 1) return TOPKV_ERR_INVALID_ARG;
  for (int32_t j = 0; j < num_layers; j += per) {
    const int32_t n = num_layers - j < per ? num_layers - j : per;
    st = topkv_internal::placed_layers_move(pack, pool, first_layer + j, n, k + j * layer_rows, cap - j * layer_rows,
                                            b.k_bytes, layer_rows, block_table, seq_len, stream);
    if (st == TOPKV_ERR_UNSUPPORTED && j == 0) break;                   // too large for the layer grid
    if (st != TOPKV_OK) return st;
  }
  if (st != TOPKV_ERR_UNSUPPORTED) return st;
  for (int32_t l = 0; l < num_layers; ++l) {                            // too large for one grid
    st = topkv_internal::placed_layers_move(pack, pool, first_layer + l, 1, k + l * layer_rows, cap - l * layer_rows,
                                            b.k_bytes, 0, block_table, seq_len, stream);
    if (st != TOPKV_OK) return st;
  }
  return TOPKV_OK;
}

// The allocation-free CRC's workspace: one copy per GPU, held until the
// process ends.  Host code never names it in a launch or a copy: the name is
// a host-side stand-in, and its device address on each device comes from
// hipGetSymbolAddress (scratch_words below).
__device__ __align__(256) uint64_t scratch[kMaxSpans];
static_assert(sizeof(scratch) == (size_t)TOPKV_CRC64_NOALLOC_SCRATCH_BYTES, "scratch size in topkv.h");

constexpr int kMaxDevices = 64;
std::atomic<uint64_t*> g_scratch[kMaxDevices];
std::mutex g_scratch_mutex;

// The current device's address of `scratch`, looked up once per device
// (with that device current) and kept.
topkv_status_t scratch_words(uint64_t** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return TOPKV_ERR_DEVICE;
  uint64_t* p = g_scratch[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    p = g_scratch[dev].load(std::memory_order_relaxed);
    if (!p) {
      void* addr = nullptr;
      if (hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch)) != hipSuccess || !addr) return TOPKV_ERR_DEVICE;
      p = static_cast<uint64_t*>(addr);
      g_scratch[dev].store(p, std::memory_order_release);
    }
  }
  *out = p;
  return TOPKV_OK;
}

}  // namespace

extern "C" {

topkv_status_t topkv_crc64_noalloc(const void* data, int64_t nbytes, uint64_t* crc_out, hipStream_t stream) {
  if (nbytes < 0 || !crc_out || (nbytes > 0 && !data)) return TOPKV_ERR_INVALID_ARG;
  if (nbytes > 0 && !aligned16(data)) return TOPKV_ERR_UNSUPPORTED;
  // every length fits: the workspace is the tables plus at most kMaxSpans span registers
  if ((int64_t)sizeof(uint64_t) * crc_words(nbytes) > (int64_t)TOPKV_CRC64_NOALLOC_SCRATCH_BYTES)
    return TOPKV_ERR_UNSUPPORTED;
  uint64_t* ws = nullptr;
  const topkv_status_t st = scratch_words(&ws);
  if (st != TOPKV_OK) return st;
  // each span kernel writes its own register before the finishing kernel
  // reads it, which reads no other word: nothing left by an earlier call is
  // read
  return crc64_launch(static_cast<const unsigned char*>(data), nbytes, finish_args(nbytes, 1, 0), ws, crc_out,
                      nullptr, nullptr, stream);
}

int64_t topkv_crc64_workspace_bytes(int64_t nbytes) {
  if (nbytes < 0) return -1;
  return (int64_t)sizeof(uint64_t) * crc_words(nbytes);
}

topkv_status_t topkv_crc64(const void* data, int64_t nbytes, void* workspace, int64_t workspace_bytes,
                           uint64_t* crc_out, hipStream_t stream) {
  if (nbytes < 0 || !crc_out || (nbytes > 0 && !data) || !workspace) return TOPKV_ERR_INVALID_ARG;
  if (workspace_bytes < topkv_crc64_workspace_bytes(nbytes)) return TOPKV_ERR_INVALID_ARG;
  if (nbytes > 0 && !aligned16(data)) return TOPKV_ERR_UNSUPPORTED;
  return crc64_launch(static_cast<const unsigned char*>(data), nbytes, finish_args(nbytes, 1, 0),
                      static_cast<uint64_t*>(workspace), crc_out, nullptr, nullptr, stream);
}

int64_t topkv_kvcache1_bytes(const topkv_pool_t* geometry, int32_t seq_len) {
  Blob b;
  return blob_geometry(geometry, seq_len, &b) == TOPKV_OK ? b.total : -1;
}

int64_t topkv_kvcache1_workspace_bytes(const topkv_pool_t* geometry, int32_t seq_len) {
  Blob b;
  return blob_geometry(geometry, seq_len, &b) == TOPKV_OK ? blob_ws_bytes(b) : -1;
}

topkv_status_t topkv_kvcache1_pack_layer(const topkv_pool_t* src, int32_t layer, const int32_t* block_table,
                                         int32_t seq_len, void* blob, int64_t blob_bytes, hipStream_t stream) {
  Blob b;
  topkv_status_t st = blob_geometry(src, seq_len, &b);
  if (st != TOPKV_OK) return st;
  if (!blob || blob_bytes < b.total || layer < 0 || layer >= src->num_layers) return TOPKV_ERR_INVALID_ARG;
  if (!aligned16(blob)) return TOPKV_ERR_UNSUPPORTED;
  if (seq_len == 0) return TOPKV_OK;
  unsigned char* k = static_cast<unsigned char*>(blob) + kHeaderBytes + (int64_t)layer * seq_len * b.row;
  return topkv_pack_layer_planes(src, layer, block_table, seq_len, k, b.k_bytes,
                                 blob_bytes - (kHeaderBytes + (int64_t)layer * seq_len * b.row), stream);
}

topkv_status_t topkv_kvcache1_seal(const topkv_pool_t* geometry, int32_t seq_len, uint64_t request_id,
                                   uint64_t model_id, void* blob, int64_t blob_bytes, void* workspace,
                                   int64_t workspace_bytes, hipStream_t stream) {
  Blob b;
  topkv_status_t st = blob_geometry(geometry, seq_len, &b);
  if (st != TOPKV_OK) return st;
  if (!blob || blob_bytes < b.total || !workspace || workspace_bytes < blob_ws_bytes(b)) return TOPKV_ERR_INVALID_ARG;
  if (!aligned16(blob)) return TOPKV_ERR_UNSUPPORTED;
  return blob_crcs(static_cast<unsigned char*>(blob), b, fields(geometry, seq_len, request_id, model_id, b),
                   kFinishSeal, nullptr, static_cast<uint64_t*>(workspace), stream);
}

topkv_status_t topkv_kvcache1_verify(const topkv_pool_t* geometry, int32_t seq_len, uint64_t request_id,
                                     uint64_t model_id, const void* blob, int64_t blob_bytes, void* workspace,
                                     int64_t workspace_bytes, int32_t* result, hipStream_t stream) {
  Blob b;
  topkv_status_t st = blob_geometry(geometry, seq_len, &b);
  if (st != TOPKV_OK) return st;
  if (!blob || blob_bytes < b.total || !workspace || workspace_bytes < blob_ws_bytes(b) || !result)
    return TOPKV_ERR_INVALID_ARG;
  if (!aligned16(blob)) return TOPKV_ERR_UNSUPPORTED;
  // (kernel 2 only reads the blob on this path: kFinishVerify writes no header)
  return blob_crcs(static_cast<unsigned char*>(const_cast<void*>(blob)), b,
                   fields(geometry, seq_len, request_id, model_id, b), kFinishVerify, result,
                   static_cast<uint64_t*>(workspace), stream);
}

topkv_status_t topkv_kvcache1_unpack_layer(const void* blob, int64_t blob_bytes, const topkv_pool_t* dst,
                                           int32_t layer, const int32_t* block_table, int32_t seq_len,
                                           hipStream_t stream) {
  Blob b;
  topkv_status_t st = blob_geometry(dst, seq_len, &b);
  if (st != TOPKV_OK) return st;
  if (!blob || blob_bytes < b.total || layer < 0 || layer >= dst->num_layers) return TOPKV_ERR_INVALID_ARG;
  if (!aligned16(blob)) return TOPKV_ERR_UNSUPPORTED;
  if (seq_len == 0) return TOPKV_OK;
  const unsigned char* k = static_cast<const unsigned char*>(blob) + kHeaderBytes + (int64_t)layer * seq_len * b.row;
  return topkv_unpack_layer_planes(k, b.k_bytes, blob_bytes - (kHeaderBytes + (int64_t)layer * seq_len * b.row),
                                   dst, layer, block_table, seq_len, stream);
}

topkv_status_t topkv_kvcache1_pack_seal(const topkv_pool_t* src, const int32_t* block_table, int32_t seq_len,
                                        uint64_t request_id, uint64_t model_id, void* blob, int64_t blob_bytes,
                                        void* workspace, int64_t workspace_bytes, hipStream_t stream) {
  Blob b;
  topkv_status_t st = blob_geometry(src, seq_len, &b);
  if (st != TOPKV_OK) return st;
  if (!src->base || !blob || blob_bytes < b.total || !workspace || workspace_bytes < blob_ws_bytes(b) ||
      (seq_len > 0 && !block_table) || src->page_size <= 0 || src->num_pages <= 0)
    return TOPKV_ERR_INVALID_ARG;
  st = topkv_internal::pool_ok(src);      // the descriptor checks of every pack/unpack, on either path
  if (st != TOPKV_OK) return st;
  if (!aligned16(blob)) return TOPKV_ERR_UNSUPPORTED;
  if (!fused_fits(src, seq_len, b)) {          // the two-step path: move every layer, then checksum
    st = kv1_move_layers(true, src, 0, src->num_layers, block_table, seq_len, blob, blob_bytes, stream);
    return st != TOPKV_OK ? st : topkv_kvcache1_seal(src, seq_len, request_id, model_id, blob, blob_bytes,
                                                      workspace, workspace_bytes, stream);
  }
  if (topkv_internal::checked_mode()) {
    st = topkv_internal::checked_tables(src, 1, block_table, (seq_len + src->page_size - 1) / src->page_size,
                                        nullptr, seq_len, 0, false, 0, 0, INT64_MAX, stream);
    if (st != TOPKV_OK) return st;
  }
  return fused_blob_crcs<kGather>(src, block_table, seq_len, static_cast<unsigned char*>(blob), b,
                                  fields(src, seq_len, request_id, model_id, b), kFinishSeal, nullptr,
                                  static_cast<uint64_t*>(workspace), stream);
}

topkv_status_t topkv_kvcache1_verify_unpack(const void* blob, int64_t blob_bytes, const topkv_pool_t* dst,
                                            const int32_t* block_table, int32_t seq_len, uint64_t request_id,
                                            uint64_t model_id, void* workspace, int64_t workspace_bytes,
                                            int32_t* result, hipStream_t stream) {
  Blob b;
  topkv_status_t st = blob_geometry(dst, seq_len, &b);
  if (st != TOPKV_OK) return st;
  if (!dst->base || !blob || blob_bytes < b.total || !workspace || workspace_bytes < blob_ws_bytes(b) || !result ||
      (seq_len > 0 && !block_table) || dst->page_size <= 0 || dst->num_pages <= 0)
    return TOPKV_ERR_INVALID_ARG;
  st = topkv_internal::pool_ok(dst);      // the descriptor checks of every pack/unpack, on either path
  if (st != TOPKV_OK) return st;
  if (!aligned16(blob)) return TOPKV_ERR_UNSUPPORTED;
  if (!fused_fits(dst, seq_len, b)) {          // the two-step path: checksum, then move every layer
    st = topkv_kvcache1_verify(dst, seq_len, request_id, model_id, blob, blob_bytes, workspace, workspace_bytes,
                               result, stream);
    return st != TOPKV_OK ? st : kv1_move_layers(false, dst, 0, dst->num_layers, block_table, seq_len,
                                                 const_cast<void*>(blob), blob_bytes, stream);
  }
  if (topkv_internal::checked_mode()) {
    st = topkv_internal::checked_tables(dst, 1, block_table, (seq_len + dst->page_size - 1) / dst->page_size,
                                        nullptr, seq_len, 0, true, 0, 0, INT64_MAX, stream);
    if (st != TOPKV_OK) return st;
  }
  return fused_blob_crcs<kScatter>(dst, block_table, seq_len, static_cast<unsigned char*>(const_cast<void*>(blob)), b,
                                   fields(dst, seq_len, request_id, model_id, b), kFinishVerify, result,
                                   static_cast<uint64_t*>(workspace), stream);
}

topkv_status_t topkv_kvcache1_pack_layers(const topkv_pool_t* src, int32_t first_layer, int32_t num_layers,
                                          const int32_t* block_table, int32_t seq_len, void* blob,
                                          int64_t blob_bytes, hipStream_t stream) {
  return kv1_move_layers(true, src, first_layer, num_layers, block_table, seq_len, blob, blob_bytes, stream);
}

topkv_status_t topkv_kvcache1_unpack_layers(const void* blob, int64_t blob_bytes, const topkv_pool_t* dst,
                                            int32_t first_layer, int32_t num_layers, const int32_t* block_table,
                                            int32_t seq_len, hipStream_t stream) {
  return kv1_move_layers(false, dst, first_layer, num_layers, block_table, seq_len, const_cast<void*>(blob),
                         blob_bytes, stream);
}

}  // extern "C"
