// Device helpers for reading and writing single codes of the packed layout
// (include/palq.h).  Used by the element-wise kernels; the convolution's
// hot loop has its own vectorised unpack.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace palq {

// Bit position of bit 2 of code jj (0..31) inside a 3-bit chunk's high word:
// codes 0-15 at the even bits, codes 16-31 at the odd bits.
__host__ __device__ inline int b3_hi_pos(int jj) {
  return 2 * (jj & 15) + (jj >> 4);
}

// Bits a code occupies in a packed row: b, except 6-bit codes, which are
// stored one per byte.
__host__ __device__ inline int store_bits(int bits) { return bits == 6 ? 8 : bits; }

__device__ inline int sext(uint32_t v, int bits) {
  const int sh = 32 - bits;
  return (int)(v << sh) >> sh;
}

// Code j of a packed row (row is 4-byte aligned).
__device__ inline int read_code(const uint8_t *row, int j, int bits, int is_signed) {
  const uint32_t *w = (const uint32_t *)row;
  uint32_t v;
  if (bits == 3) {
    const uint32_t *ch = w + 3 * (j >> 5);
    const int jj = j & 31;
    v = (ch[jj >> 4] >> (2 * (jj & 15))) & 3u;
    v |= ((ch[2] >> b3_hi_pos(jj)) & 1u) << 2;
  } else {
    const int bit = j * store_bits(bits);
    v = (w[bit >> 5] >> (bit & 31)) & ((1u << bits) - 1u);
  }
  return is_signed ? sext(v, bits) : (int)v;
}

// Packs up to 32 codes (c[0..ncodes), the rest taken as 0) of one 32-code
// chunk into its words; returns the number of words of the chunk
// (bits words for b in {2,4,8}, 8 for b = 6 (one code per byte), 3 for
// b = 3).
__device__ inline int pack_chunk(const int *c, int ncodes, int bits, uint32_t *words) {
  if (bits == 3) {
    uint32_t lo0 = 0, lo1 = 0, hi = 0;
    for (int j = 0; j < 32; ++j) {
      const uint32_t v = j < ncodes ? (uint32_t)c[j] & 7u : 0u;
      if (j < 16) lo0 |= (v & 3u) << (2 * j);
      else lo1 |= (v & 3u) << (2 * (j - 16));
      hi |= ((v >> 2) & 1u) << b3_hi_pos(j);
    }
    words[0] = lo0; words[1] = lo1; words[2] = hi;
    return 3;
  }
  const int sb = store_bits(bits);
  const int per = 32 / sb;
  const uint32_t mask = (1u << bits) - 1u;
  for (int wi = 0; wi < sb; ++wi) {
    uint32_t acc = 0;
    for (int k = 0; k < per; ++k) {
      const int j = wi * per + k;
      const uint32_t v = j < ncodes ? (uint32_t)c[j] & mask : 0u;
      acc |= v << (k * sb);
    }
    words[wi] = acc;
  }
  return sb;
}

// Words of chunk `ci` that lie inside a row of `row_words` words.
__device__ inline int chunk_words_in_row(int ci, int bits, int64_t row_words) {
  const int per_chunk = bits == 3 ? 3 : store_bits(bits);
  int64_t left = row_words - (int64_t)ci * per_chunk;
  return left < per_chunk ? (int)left : per_chunk;
}

}  // namespace palq
