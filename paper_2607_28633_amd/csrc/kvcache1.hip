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
// ~(~0 * x^(8N) + R(data)).  Work split:
//   kernel 0: byte tables into the caller's workspace (slicing-by-8, and
//     multiply-by-constant tables for the two fixed shifts below);
//   kernel 1: each workgroup owns a 256 KiB chunk = 16 sub-chunks of 16 KiB;
//     lane t takes bytes [64t, 64t + 64) of every sub-chunk (adjacent loads),
//     runs them through the slicing tables (in LDS), advances its running
//     register by one sub-chunk per step with a table multiply, and a tree
//     of shift-and-add steps joins the lanes.  The data is front-padded with
//     zero bytes to whole chunks (free, by the property above);
//   kernel 2: one workgroup folds the chunk values (each lane a run of 2^q
//     chunks, then a tree), appends the sub-16-byte tail and applies the
//     preset and complement.
// Shift constants x^(8 * 2^k) mod P are computed once on the host.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstring>

#include "topkv.h"

namespace {

constexpr uint64_t kPolyReflected = 0xC96C5795D7870F42ull;   // ECMA-182, bit-reversed
constexpr int kCrcThreads = 256;
constexpr int kPiece = 64;                                      // bytes per lane per sub-chunk
constexpr int kSubLog2 = 14;                                    // 16 KiB sub-chunk = 256 lanes x 64 B
constexpr int kSubs = 16;                                       // sub-chunks per workgroup
constexpr int kChunkLog2 = 18;                                  // 256 KiB per workgroup
constexpr int64_t kChunk = (int64_t)1 << kChunkLog2;
constexpr int kTableWords = 8 * 256;                            // one set of 8 byte tables
// workspace: [slicing tables][x^(8*16K) tables][x^(8*256K) tables][chunk registers...]
constexpr int64_t kWsTables = 3 * kTableWords;

struct ShiftConsts {
  uint64_t x8pow2[64];    // x^(8 * 2^k) mod P, reflected
};

__host__ __device__ inline uint64_t mul_x(uint64_t w) { return (w >> 1) ^ ((w & 1) ? kPolyReflected : 0); }

// a * b mod P in the reflected representation (bit 63 of a is its x^0 term).
__host__ __device__ inline uint64_t mulmod(uint64_t a, uint64_t b) {
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

// Kernel 0: the byte tables every other kernel copies into LDS.
//   [0, 2048):     slicing-by-8, t[k][b] = byte b followed by k zero bytes
//   [2048, 4096):  b << 8k times x^(8 * 16 KiB)   (advance one sub-chunk)
//   [4096, 6144):  b << 8k times x^(8 * 256 KiB)  (advance one chunk)
// Multiplying a register by a constant is linear, so it is the XOR of one
// lookup per register byte in such a table.
__global__ __launch_bounds__(256) void crc64_tables_kernel(uint64_t* __restrict__ tables, uint64_t sub_shift,
                                                           uint64_t chunk_shift) {
  const int g = blockIdx.x * 256 + threadIdx.x;              // grid covers exactly 3 * 2048 entries
  const int set = g / kTableWords, k = (g / 256) % 8, b = g % 256;
  uint64_t v;
  if (set == 0) {
    v = (uint64_t)b;
    for (int i = 0; i < 8 * (k + 1); ++i) v = mul_x(v);
  } else {
    v = mulmod((uint64_t)b << (8 * k), set == 1 ? sub_shift : chunk_shift);
  }
  tables[g] = v;
}

__device__ inline uint64_t lookup8(uint64_t v, const uint64_t* t) {   // t: 8 x 256 words
  return t[0 * 256 + (v & 0xff)] ^ t[1 * 256 + ((v >> 8) & 0xff)] ^ t[2 * 256 + ((v >> 16) & 0xff)] ^
         t[3 * 256 + ((v >> 24) & 0xff)] ^ t[4 * 256 + ((v >> 32) & 0xff)] ^ t[5 * 256 + ((v >> 40) & 0xff)] ^
         t[6 * 256 + ((v >> 48) & 0xff)] ^ t[7 * 256 + (v >> 56)];
}

// Eight bytes (little-endian word w) into the register: with the slicing
// tables, byte 0 is followed by 7 more bytes, byte 7 by none.
__device__ inline uint64_t crc_word(uint64_t reg, uint64_t w, const uint64_t* t) {
  reg ^= w;
  return t[7 * 256 + (reg & 0xff)] ^ t[6 * 256 + ((reg >> 8) & 0xff)] ^ t[5 * 256 + ((reg >> 16) & 0xff)] ^
         t[4 * 256 + ((reg >> 24) & 0xff)] ^ t[3 * 256 + ((reg >> 32) & 0xff)] ^
         t[2 * 256 + ((reg >> 40) & 0xff)] ^ t[1 * 256 + ((reg >> 48) & 0xff)] ^ t[0 * 256 + (reg >> 56)];
}

__device__ inline void copy_words(uint64_t* lds, const uint64_t* __restrict__ src, int words) {
  for (int i = threadIdx.x; i < words; i += blockDim.x) lds[i] = src[i];
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Kernel 1: raw register of each 256 KiB chunk of the front-padded stream.
// data: 16-byte aligned, `head` bytes (a multiple of 16); `pad` leading zero
// bytes (a multiple of 16) make head + pad a whole number of chunks.  Lane t
// owns bytes [t*64, t*64 + 64) of each 16 KiB sub-chunk (four adjacent
// 16-byte loads, so every line is used at once), folds its pieces across the
// 16 sub-chunks (advance by 16 KiB = one table multiply), and a tree of
// shift-and-add steps joins the 256 lanes.
__global__ __launch_bounds__(kCrcThreads) void crc64_chunks_kernel(const u32x4* __restrict__ data, int64_t head,
                                                                   int64_t pad, const uint64_t* __restrict__ tables,
                                                                   uint64_t* __restrict__ partial, ShiftConsts sc) {
  __shared__ uint64_t t_slice[kTableWords];
  __shared__ uint64_t t_sub[kTableWords];
  __shared__ uint64_t acc[kCrcThreads];
  copy_words(t_slice, tables, kTableWords);
  copy_words(t_sub, tables + kTableWords, kTableWords);
  __syncthreads();
  const int64_t base = (int64_t)blockIdx.x * kChunk + (int64_t)threadIdx.x * kPiece - pad;   // data offset
  u32x4 cur[4], nxt[4];
  auto load = [&](u32x4 (&v)[4], int sub) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t off = base + ((int64_t)sub << kSubLog2) + 16 * j;
      v[j] = off >= 0 ? __builtin_nontemporal_load(data + off / 16) : u32x4{0u, 0u, 0u, 0u};   // off < head
    }
  };
  load(cur, 0);
  uint64_t fold = 0;
#pragma unroll 2
  for (int sub = 0; sub < kSubs; ++sub) {
    if (sub + 1 < kSubs) load(nxt, sub + 1);
    uint64_t reg = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      reg = crc_word(reg, ((uint64_t)cur[j].y << 32) | cur[j].x, t_slice);
      reg = crc_word(reg, ((uint64_t)cur[j].w << 32) | cur[j].z, t_slice);
    }
    fold = lookup8(fold, t_sub) ^ reg;
#pragma unroll
    for (int j = 0; j < 4; ++j) cur[j] = nxt[j];
  }
  acc[threadIdx.x] = fold;
  __syncthreads();
  // join lanes t and t + s: the later group holds s lanes x 64 bytes of every sub-chunk
  for (int lvl = 0; lvl < 8; ++lvl) {
    const int s = 1 << lvl;
    const int t = threadIdx.x;
    if ((t & (2 * s - 1)) == 0) acc[t] = mulmod(sc.x8pow2[6 + lvl], acc[t]) ^ acc[t + s];
    __syncthreads();
  }
  if (threadIdx.x == 0) partial[blockIdx.x] = acc[0];
}

// Kernel 2 (one workgroup): fold `chunks` chunk registers, each lane a run of
// 2^run_log2 of them (front-padded with zero registers; advancing one chunk is
// one table multiply), join the lanes, append the tail bytes and finish:
// out = ~(preset_shift + R).
__global__ __launch_bounds__(kCrcThreads) void crc64_finish_kernel(const uint64_t* __restrict__ tables,
                                                                   const uint64_t* __restrict__ partial,
                                                                   int64_t chunks, int run_log2,
                                                                   const unsigned char* __restrict__ tail,
                                                                   int tail_len, uint64_t preset_shift,
                                                                   uint64_t* __restrict__ out, ShiftConsts sc) {
  __shared__ uint64_t t_chunk[kTableWords];
  __shared__ uint64_t acc[kCrcThreads];
  copy_words(t_chunk, tables + 2 * kTableWords, kTableWords);
  __syncthreads();
  const int64_t run = (int64_t)1 << run_log2;
  const int64_t lead = (int64_t)kCrcThreads * run - chunks;    // leading zero chunks
  uint64_t reg = 0;
  for (int64_t j0 = 0; j0 < run; j0 += 8) {
    uint64_t vals[8];   // issue the loads of eight chunk registers, then fold them
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int64_t v = (int64_t)threadIdx.x * run + j0 + j - lead;
      vals[j] = (j0 + j < run && v >= 0) ? partial[v] : 0ull;
    }
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (j0 + j < run) reg = lookup8(reg, t_chunk) ^ vals[j];
  }
  acc[threadIdx.x] = reg;
  __syncthreads();
  for (int lvl = 0; lvl < 8; ++lvl) {
    const int s = 1 << lvl;
    const int t = threadIdx.x;
    if ((t & (2 * s - 1)) == 0) acc[t] = mulmod(sc.x8pow2[kChunkLog2 + run_log2 + lvl], acc[t]) ^ acc[t + s];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    uint64_t r = acc[0];
    for (int b = 0; b < tail_len; ++b) r = tables[(r ^ tail[b]) & 0xff] ^ (r >> 8);   // slicing table 0
    out[0] = ~(preset_shift ^ r);
  }
}

int64_t crc_chunks(int64_t head) { return (head + kChunk - 1) / kChunk; }

// Workspace words one CRC of n bytes needs: tables + chunk registers.
int64_t crc_words(int64_t n) { return kWsTables + crc_chunks(n - n % 16) + 1; }

// Queue the byte tables into ws (first kWsTables words).
topkv_status_t crc64_tables(uint64_t* ws, hipStream_t stream) {
  const ShiftConsts& sc = shift_consts();
  hipLaunchKernelGGL(crc64_tables_kernel, dim3((unsigned)(kWsTables / 256)), dim3(256), 0, stream, ws,
                     sc.x8pow2[kSubLog2], sc.x8pow2[kChunkLog2]);
  return hipGetLastError() == hipSuccess ? TOPKV_OK : TOPKV_ERR_LAUNCH;
}

// Queue the CRC-64/XZ of data[0, n) into out (device).  data 16-byte aligned;
// ws holds the tables (crc64_tables) followed by room for the chunk registers.
topkv_status_t crc64_launch(const unsigned char* data, int64_t n, const uint64_t* tables, uint64_t* partial,
                            uint64_t* out, hipStream_t stream) {
  const ShiftConsts& sc = shift_consts();
  const int64_t head = n - n % 16;
  const int64_t chunks = crc_chunks(head);
  const int64_t pad = chunks * kChunk - head;
  if (chunks > 0) {
    if (chunks > INT32_MAX) return TOPKV_ERR_UNSUPPORTED;
    hipLaunchKernelGGL(crc64_chunks_kernel, dim3((unsigned)chunks), dim3(kCrcThreads), 0, stream,
                       reinterpret_cast<const u32x4*>(data), head, pad, tables, partial, sc);
    if (hipGetLastError() != hipSuccess) return TOPKV_ERR_LAUNCH;
  }
  int run_log2 = 0;
  while (((int64_t)kCrcThreads << run_log2) < chunks) ++run_log2;
  if (kChunkLog2 + run_log2 + 8 > 63) return TOPKV_ERR_UNSUPPORTED;
  hipLaunchKernelGGL(crc64_finish_kernel, dim3(1), dim3(kCrcThreads), 0, stream, tables, partial, chunks, run_log2,
                     data + head, (int)(n - head), mulmod(x8n(sc, (uint64_t)n), ~0ull), out, sc);
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
      __builtin_mul_overflow(row * seq_len, (int64_t)g->num_layers, &tensor))
    return TOPKV_ERR_UNSUPPORTED;
  if (row % 16) return TOPKV_ERR_UNSUPPORTED;   // tensors must stay 16-byte aligned inside the blob
  b->row = row;
  b->k_bytes = tensor;
  b->v_bytes = g->planes == 2 ? tensor : 0;
  b->total = kHeaderBytes + b->k_bytes + b->v_bytes;
  return TOPKV_OK;
}

struct HeaderFields {
  uint64_t request_id, model_id;
  uint32_t seq_len, layers, kv_heads, head_dim, elem_bytes, planes;
  uint64_t k_bytes, v_bytes;
};

// Writes the 128-byte header: 16 lanes each store one little-endian 8-byte
// word (vector stores); words 8 and 9 are the two checksums from `crcs`.
__global__ void kv1_header_kernel(unsigned char* __restrict__ blob, HeaderFields f,
                                  const uint64_t* __restrict__ crcs) {
  const int w = threadIdx.x;
  if (w >= 16) return;
  uint64_t v = 0;
  switch (w) {
    case 0: memcpy(&v, "KVCACHE1", 8); break;
    case 1: v = f.request_id; break;
    case 2: v = f.model_id; break;
    case 3: v = (uint64_t)f.seq_len | ((uint64_t)f.layers << 32); break;
    case 4: v = (uint64_t)f.kv_heads | ((uint64_t)f.head_dim << 32); break;
    case 5: v = (uint64_t)f.elem_bytes | ((uint64_t)f.planes << 32); break;
    case 6: v = f.k_bytes; break;
    case 7: v = f.v_bytes; break;
    case 8: v = crcs[0]; break;
    case 9: v = crcs[1]; break;
    default: v = 0; break;
  }
  reinterpret_cast<uint64_t*>(blob)[w] = v;
}

// result[0] status, [1] header fields differing from the expected geometry
// (bit mask over header words 0-7), [2] K checksum mismatch, [3] V mismatch.
__global__ void kv1_verify_kernel(const unsigned char* __restrict__ blob, HeaderFields f,
                                  const uint64_t* __restrict__ crcs, int32_t* __restrict__ result) {
  if (threadIdx.x != 0) return;
  const uint64_t* h = reinterpret_cast<const uint64_t*>(blob);
  uint64_t magic;
  memcpy(&magic, "KVCACHE1", 8);
  const uint64_t want[8] = {magic, f.request_id, f.model_id, (uint64_t)f.seq_len | ((uint64_t)f.layers << 32),
                            (uint64_t)f.kv_heads | ((uint64_t)f.head_dim << 32),
                            (uint64_t)f.elem_bytes | ((uint64_t)f.planes << 32), f.k_bytes, f.v_bytes};
  int32_t bad = 0;
  for (int w = 0; w < 8; ++w)
    if (h[w] != want[w]) bad |= 1 << w;
  const int32_t ck = h[8] != crcs[0];
  const int32_t cv = h[9] != crcs[1];
  result[0] = (bad | ck | cv) ? (int32_t)TOPKV_ERR_CHECKSUM : (int32_t)TOPKV_OK;
  result[1] = bad;
  result[2] = ck;
  result[3] = cv;
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

// Both checksums of a blob body into ws[0..1]; then the byte tables, then
// the chunk registers of K and of V.
topkv_status_t blob_crcs(const unsigned char* blob, const Blob& b, uint64_t* ws, hipStream_t stream) {
  uint64_t* tables = ws + 2;
  uint64_t* partial_k = tables + kWsTables;
  uint64_t* partial_v = partial_k + crc_words(b.k_bytes) - kWsTables;
  topkv_status_t st = crc64_tables(tables, stream);
  if (st != TOPKV_OK) return st;
  st = crc64_launch(blob + kHeaderBytes, b.k_bytes, tables, partial_k, ws, stream);
  if (st != TOPKV_OK) return st;
  return crc64_launch(blob + kHeaderBytes + b.k_bytes, b.v_bytes, tables, partial_v, ws + 1, stream);
}

int64_t blob_ws_bytes(const Blob& b) {
  return (int64_t)sizeof(uint64_t) * (2 + crc_words(b.k_bytes) + crc_words(b.v_bytes) - kWsTables);
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

}  // namespace

extern "C" {

int64_t topkv_crc64_workspace_bytes(int64_t nbytes) {
  if (nbytes < 0) return -1;
  return (int64_t)sizeof(uint64_t) * crc_words(nbytes);
}

topkv_status_t topkv_crc64(const void* data, int64_t nbytes, void* workspace, int64_t workspace_bytes,
                           uint64_t* crc_out, hipStream_t stream) {
  if (nbytes < 0 || !crc_out || (nbytes > 0 && !data) || !workspace) return TOPKV_ERR_INVALID_ARG;
  if (workspace_bytes < topkv_crc64_workspace_bytes(nbytes)) return TOPKV_ERR_INVALID_ARG;
  if (nbytes > 0 && !aligned16(data)) return TOPKV_ERR_UNSUPPORTED;
  uint64_t* ws = static_cast<uint64_t*>(workspace);
  const topkv_status_t st = crc64_tables(ws, stream);
  if (st != TOPKV_OK) return st;
  return crc64_launch(static_cast<const unsigned char*>(data), nbytes, ws, ws + kWsTables, crc_out, stream);
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
  uint64_t* ws = static_cast<uint64_t*>(workspace);
  unsigned char* bytes = static_cast<unsigned char*>(blob);
  st = blob_crcs(bytes, b, ws, stream);
  if (st != TOPKV_OK) return st;
  hipLaunchKernelGGL(kv1_header_kernel, dim3(1), dim3(64), 0, stream, bytes,
                     fields(geometry, seq_len, request_id, model_id, b), (const uint64_t*)ws);
  return hipGetLastError() == hipSuccess ? TOPKV_OK : TOPKV_ERR_LAUNCH;
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
  uint64_t* ws = static_cast<uint64_t*>(workspace);
  const unsigned char* bytes = static_cast<const unsigned char*>(blob);
  st = blob_crcs(bytes, b, ws, stream);
  if (st != TOPKV_OK) return st;
  hipLaunchKernelGGL(kv1_verify_kernel, dim3(1), dim3(64), 0, stream, bytes,
                     fields(geometry, seq_len, request_id, model_id, b), (const uint64_t*)ws, result);
  return hipGetLastError() == hipSuccess ? TOPKV_OK : TOPKV_ERR_LAUNCH;
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

}  // extern "C"
