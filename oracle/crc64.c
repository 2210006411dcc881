/* oracle/crc64.c - CRC-64/XZ, one byte at a time.  TEST INFRASTRUCTURE ONLY
 * (the CPU oracle; never linked into the product library).
 *
 * The KV cache serialization format (arxiv 2607.28633, Section 3.5) carries a
 * CRC-64 of the key tensor and of the value tensor; the paper does not name
 * the polynomial.  This oracle uses CRC-64/XZ: the ECMA-182 polynomial
 * 0x42F0E1EBA9EA3693 in reflected (LSB-first) form 0xC96C5795D7870F42,
 * register preset to all ones, result complemented.  The table is built from
 * the polynomial: entry i is the register after shifting byte i in.
 */
#include <stddef.h>
#include <stdint.h>

static const uint64_t kPolyReflected = 0xC96C5795D7870F42ull;
static uint64_t table[256];

__attribute__((constructor)) static void build_table(void) {
  for (int i = 0; i < 256; ++i) {
    uint64_t c = (uint64_t)i;
    for (int k = 0; k < 8; ++k) c = (c & 1) ? (c >> 1) ^ kPolyReflected : c >> 1;
    table[i] = c;
  }
}

/* Continue a CRC over n more bytes: oracle_crc64_update(oracle_crc64_update(0, a), b)
 * equals the CRC of a followed by b; oracle_crc64_update(0, p, n) is the CRC of p. */
uint64_t oracle_crc64_update(uint64_t crc, const uint8_t* p, size_t n) {
  uint64_t reg = ~crc;
  for (size_t i = 0; i < n; ++i) reg = table[(reg ^ p[i]) & 0xff] ^ (reg >> 8);
  return ~reg;
}
