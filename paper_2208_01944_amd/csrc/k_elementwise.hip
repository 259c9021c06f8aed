// Element-wise and reduction kernels of the PalQuant path: pack/unpack,
// the Eq. 2 quantiser with its min/max calibration, the standalone cyclic
// permutation (Eq. 8), max pool, integer global sum and the FC layer.
// All are bandwidth-bound; one thread handles one 32-code chunk of a row so
// that every packed word is written by exactly one thread.
#include <float.h>
#include <math.h>
#include <stdlib.h>

#include "codes.h"

#include <algorithm>

#include "palq_internal.h"

namespace palq {

namespace {

constexpr int kBlock = 256;

inline unsigned grid_for(int64_t items) {
  int64_t g = (items + kBlock - 1) / kBlock;
  return (unsigned)(g < 1 ? 1 : g);
}

// ------------------------------------------------------------ pack/unpack
__global__ void pack_kernel(const uint8_t *codes, ActView out, int64_t rows, int chunks) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= rows * chunks) return;
  const int64_t r = t / chunks;      // (pixel, group) row
  const int ci = (int)(t % chunks);  // chunk of 32 codes
  const int j0 = ci * 32;
  const int nc = min(32, out.cpg - j0);
  int c[32];
  const uint8_t *src = codes + r * out.cpg + j0;
  for (int j = 0; j < 32; ++j) c[j] = j < nc ? (int)src[j] : 0;
  uint32_t words[8];
  pack_chunk(c, nc, out.bits, words);
  const int per_chunk = out.bits == 3 ? 3 : store_bits(out.bits);
  const int nw = chunk_words_in_row(ci, out.bits, out.row / 4);
  uint32_t *dst = (uint32_t *)row_at(out, r) + (int64_t)ci * per_chunk;
  for (int k = 0; k < nw; ++k) dst[k] = words[k];
}

__global__ void unpack_kernel(ActView in, uint8_t *codes, int64_t rows, int chunks) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= rows * chunks) return;
  const int64_t r = t / chunks;
  const int ci = (int)(t % chunks);
  const int j0 = ci * 32;
  const int nc = min(32, in.cpg - j0);
  const uint8_t *row = row_at(in, r);
  uint8_t *dst = codes + r * in.cpg + j0;
  for (int j = 0; j < nc; ++j) dst[j] = (uint8_t)read_code(row, j0 + j, in.bits, in.is_signed);
}

// ------------------------------------------------------------ quantiser
// Order-preserving map of fp32 to uint32 for atomic min/max.
__device__ inline uint32_t f2ord(float f) {
  const uint32_t b = __float_as_uint(f);
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}
__device__ inline float ord2f(uint32_t o) {
  return __uint_as_float((o & 0x80000000u) ? (o & 0x7fffffffu) : ~o);
}

__global__ void range_init_kernel(uint32_t *enc) {
  enc[0] = 0xffffffffu;  // running min
  enc[1] = 0u;           // running max
}

__global__ void minmax_kernel(const float *x, int64_t count, uint32_t *enc) {
  uint32_t lo = 0xffffffffu, hi = 0u;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count;
       i += (int64_t)gridDim.x * blockDim.x) {
    const float v = x[i];
    if (v == v) {  // skip NaN
      const uint32_t o = f2ord(v);
      lo = min(lo, o);
      hi = max(hi, o);
    }
  }
  // wave64 reduction, then one atomic per wave (min/max are order-free)
  for (int off = 32; off > 0; off >>= 1) {
    lo = min(lo, (uint32_t)__shfl_xor((int)lo, off));
    hi = max(hi, (uint32_t)__shfl_xor((int)hi, off));
  }
  if ((threadIdx.x & 63) == 0) {
    atomicMin(&enc[0], lo);
    atomicMax(&enc[1], hi);
  }
}

__global__ void range_out_kernel(const uint32_t *enc, float *range_out) {
  const bool empty = enc[0] == 0xffffffffu && enc[1] == 0u;
  range_out[0] = empty ? __uint_as_float(0x7fc00000u) : ord2f(enc[0]);
  range_out[1] = empty ? __uint_as_float(0x7fc00000u) : ord2f(enc[1]);
}

// Eq. 2 in the documented fp32 op order, for one code.
__device__ inline int quant_one(float x, float l, float rng, float qmax) {
  const float d = x - l;
  float t = d / rng;  // correctly rounded (built with correctly rounded division)
  t = t > 1.0f ? 1.0f : t;
  t = t >= 0.0f ? t : 0.0f;
  return (int)rintf(t * qmax);
}

// 8-bit codes of 3-channel pixels (one 4-byte row each, the image input):
// one thread per 4 pixels, three 16-byte loads and one 16-byte store.
__global__ void quantize_px3_kernel(const float *x, float l, float u, const uint32_t *enc, ActView out,
                                    int64_t quads) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= quads) return;
  bool degenerate = false;
  if (enc) {
    const bool empty = enc[0] == 0xffffffffu && enc[1] == 0u;
    l = ord2f(enc[0]);
    u = ord2f(enc[1]);
    degenerate = empty || !(u > l);
  }
  const float rng = u - l;
  const int off = out.is_signed ? 128 : 0;
  const float4 *src = (const float4 *)(x + 12 * t);
  const float4 f0 = src[0], f1 = src[1], f2 = src[2];
  const float v[12] = {f0.x, f0.y, f0.z, f0.w, f1.x, f1.y, f1.z, f1.w, f2.x, f2.y, f2.z, f2.w};
  uint32_t w[4];
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    uint32_t word = 0;
#pragma unroll
    for (int c = 0; c < 3; ++c) {
      const int q = (degenerate ? 0 : quant_one(v[3 * p + c], l, rng, 255.0f)) - off;
      word |= ((uint32_t)q & 0xffu) << (8 * c);
    }
    w[p] = word;
  }
  *(uint4 *)(out.data + 16 * t) = make_uint4(w[0], w[1], w[2], w[3]);
}

// Signed 8-bit codes of 3-channel fp32 pixels written straight into a
// copy with a `pad`-pixel zero border (4-byte pixel rows): kQPadRows output
// rows per workgroup, one column per thread, every row's loads issued
// before any store.  Same arithmetic as quantize_px3_kernel.
constexpr int kQPadRows = 8;
__global__ void quantize_pad_kernel(const float *x, float l, float u, int in_h, int in_w, int pad, ActView out,
                                    int rows) {
  const int r0 = (int)blockIdx.x * kQPadRows;
  const float rng = u - l;
  for (int c = threadIdx.x; c < out.w; c += blockDim.x) {
    const int ix = c - pad;
    float v[kQPadRows][3];
    bool in[kQPadRows];
#pragma unroll
    for (int j = 0; j < kQPadRows; ++j) {
      const int r = r0 + j, y = r % out.h, n = r / out.h, iy = y - pad;
      in[j] = r < rows && iy >= 0 && iy < in_h && ix >= 0 && ix < in_w;
      const float *src = x + (((int64_t)n * in_h + (in[j] ? iy : 0)) * in_w + (in[j] ? ix : 0)) * 3;
#pragma unroll
      for (int ch = 0; ch < 3; ++ch) v[j][ch] = in[j] ? src[ch] : 0.0f;
    }
#pragma unroll
    for (int j = 0; j < kQPadRows; ++j) {
      if (r0 + j >= rows) break;
      uint32_t word = 0;
      if (in[j]) {
#pragma unroll
        for (int ch = 0; ch < 3; ++ch) word |= ((uint32_t)(quant_one(v[j][ch], l, rng, 255.0f) - 128) & 0xffu) << (8 * ch);
      }
      ((uint32_t *)(out.data + ((int64_t)(r0 + j) * out.w + c) * out.pixel))[0] = word;
    }
  }
}

// The same with four input pixels per thread (three 16-byte loads) for
// rows of at most 4 (64 - 2 pad) pixels, in_w % 4 == 0: 64 threads per
// output row (quads of interior pixels, then the 2 pad border pixels), four
// rows per workgroup; border rows are zeroed by all 64.
__global__ void quantize_pad4_kernel(const float *x, float l, float u, int in_h, int in_w, int pad, ActView out,
                                     int rows) {
  const int r = (int)blockIdx.x * 4 + (int)(threadIdx.x >> 6), j = (int)(threadIdx.x & 63);
  if (r >= rows) return;
  const int y = r % out.h, n = r / out.h, iy = y - pad;
  uint32_t *row = (uint32_t *)(out.data + (int64_t)r * out.w * out.pixel);
  if (iy < 0 || iy >= in_h) {
    for (int c = j; c < out.w; c += 64) row[c] = 0u;
    return;
  }
  const int quads = in_w >> 2;
  if (j < quads) {
    const float4 *src = (const float4 *)(x + (((int64_t)n * in_h + iy) * in_w + 4 * j) * 3);
    const float4 f0 = src[0], f1 = src[1], f2 = src[2];
    const float v[12] = {f0.x, f0.y, f0.z, f0.w, f1.x, f1.y, f1.z, f1.w, f2.x, f2.y, f2.z, f2.w};
    const float rng = u - l;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      uint32_t word = 0;
#pragma unroll
      for (int ch = 0; ch < 3; ++ch) word |= ((uint32_t)(quant_one(v[3 * p + ch], l, rng, 255.0f) - 128) & 0xffu) << (8 * ch);
      row[pad + 4 * j + p] = word;
    }
  } else if (j - quads < 2 * pad) {
    const int b = j - quads;
    row[b < pad ? b : in_w + b] = 0u;
  }
}

// One thread per packed word (b in {2, 4, 8}) or 32-code chunk (b = 3).
__global__ void quantize_kernel(const float *x, float l, float u, const uint32_t *enc, ActView out,
                                int64_t rows, int units) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= rows * units) return;
  bool degenerate = false;
  if (enc) {
    const bool empty = enc[0] == 0xffffffffu && enc[1] == 0u;
    l = ord2f(enc[0]);
    u = ord2f(enc[1]);
    degenerate = empty || !(u > l);
  }
  const int64_t r = t / units;
  const int wi = (int)(t % units);
  const float qmax = (float)((1 << out.bits) - 1);
  const float rng = u - l;
  const int off = out.is_signed ? (1 << (out.bits - 1)) : 0;
  const float *src = x + r * out.cpg;
  uint32_t *dst = (uint32_t *)row_at(out, r);
  if (out.bits == 3) {
    int c[32];
    const int j0 = wi * 32;
    const int nc = min(32, out.cpg - j0);
    for (int j = 0; j < 32; ++j)
      c[j] = (j < nc && !degenerate ? quant_one(src[j0 + j], l, rng, qmax) : 0) - off;
    uint32_t words[3];
    pack_chunk(c, nc, 3, words);
    dst[3 * wi] = words[0];
    dst[3 * wi + 1] = words[1];
    dst[3 * wi + 2] = words[2];
    return;
  }
  const int per = 32 / store_bits(out.bits);
  const int j0 = wi * per;
  const int nc = min(per, out.cpg - j0);
  const uint32_t mask = (1u << out.bits) - 1u;
  uint32_t w = 0;
  for (int k = 0; k < nc; ++k) {
    const int q = (degenerate ? 0 : quant_one(src[j0 + k], l, rng, qmax)) - off;
    w |= ((uint32_t)q & mask) << (k * store_bits(out.bits));
  }
  dst[wi] = w;
}

// ------------------------------------------------------------ shuffle (Eq. 8)
__global__ void shuffle_kernel(ActView in, int steps, ActView out, int64_t pixels) {
  const int64_t words = in.row / 4;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t per_pixel = (int64_t)in.groups * words;
  if (t >= pixels * per_pixel) return;
  const int64_t p = t / per_pixel;
  const int64_t rem = t % per_pixel;
  const int g = (int)(rem / words);
  const int64_t wi = rem % words;
  const int gd = (g + steps) % in.groups;
  const uint32_t *src = (const uint32_t *)(in.data + p * in.pixel + g * in.gstride);
  uint32_t *dst = (uint32_t *)(out.data + p * out.pixel + gd * out.gstride);
  dst[wi] = src[wi];
}

// ------------------------------------------------------------ channel shuffle
// Channel shuffle across the G groups of a pixel (the [G][C] channel matrix
// transposed to [C][G]): output channel o = g' C + c' takes input channel
// (o mod G) C + o / G.  One thread per output 32-code chunk.
__global__ void channel_shuffle_kernel(ActView in, ActView out, int64_t pixels, int chunks) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t per_pixel = (int64_t)out.groups * chunks;
  if (t >= pixels * per_pixel) return;
  const int64_t p = t / per_pixel;
  const int rem = (int)(t % per_pixel);
  const int gq = rem / chunks, ci = rem % chunks;
  const int C = out.cpg, G = out.groups;
  const uint8_t *src = in.data + p * in.pixel;
  const int n = min(32, C - ci * 32);
  int c[32];
  for (int j = 0; j < 32; ++j) {
    if (j < n) {
      const int o = gq * C + ci * 32 + j;
      c[j] = read_code(src + (int64_t)(o % G) * in.gstride, o / G, in.bits, in.is_signed);
    } else {
      c[j] = 0;
    }
  }
  uint32_t words[8];
  pack_chunk(c, n, out.bits, words);
  uint32_t *dst = (uint32_t *)(out.data + p * out.pixel + (int64_t)gq * out.gstride) + (int64_t)ci * (out.bits == 3 ? 3 : store_bits(out.bits));
  const int nw = chunk_words_in_row(ci, out.bits, out.row / 4);
  for (int wi = 0; wi < nw; ++wi) dst[wi] = words[wi];
}

// Unpadded rows of b in {2, 4, 8} with G a power of two up to 16: the
// output's flat code o = 4F t + f (F codes per word, thread t) takes code
// (4F t + f) / G of group f mod G, so each group hands a thread one aligned
// run of 128 / G bits and the G runs interleave field by field into four
// whole output words, written with one 16-byte store.
template <int B, int G>
__global__ void channel_shuffle_words_kernel(ActView in, ActView out, int64_t threads, int tpp) {
  constexpr int F = 32 / B;      // codes per word
  constexpr int GB = 128 / G;    // bits each group hands a thread
  constexpr int NW = GB >= 32 ? GB / 32 : 1;
  constexpr uint32_t mask = (1u << B) - 1u;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= threads) return;
  const int64_t p = t / tpp;
  const int tl = (int)(t - p * tpp);
  const uint8_t *src = in.data + p * in.pixel;
  uint32_t s[G][NW];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const uint32_t *r = (const uint32_t *)(src + (int64_t)g * in.gstride);
    if constexpr (GB >= 32) {
#pragma unroll
      for (int j = 0; j < NW; ++j) s[g][j] = r[tl * NW + j];
    } else {
      constexpr int PER = 32 / GB;
      s[g][0] = r[tl / PER] >> ((tl % PER) * GB);
    }
  }
  uint32_t o[4] = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int f = 0; f < 4 * F; ++f) {
    const int g = f % G, i = f / G;
    const uint32_t v = (s[g][(i * B) / 32] >> ((i * B) % 32)) & mask;
    o[f / F] |= v << ((f % F) * B);
  }
  // bytes 16 tl .. of the pixel's G rows: row gq, 16-byte aligned inside it
  const int b = 16 * tl, gq = b / (int)out.row;
  *(uint4 *)(out.data + p * out.pixel + gq * out.gstride + (b - gq * (int)out.row)) =
      make_uint4(o[0], o[1], o[2], o[3]);
}

// ------------------------------------------------------------ max pool
// Field-wise max of sixteen 2-bit unsigned fields packed in a word.
__device__ inline uint32_t max2x16(uint32_t a, uint32_t b) {
  const uint32_t L = 0x55555555u;
  const uint32_t a1 = (a >> 1) & L, a0 = a & L, b1 = (b >> 1) & L, b0 = b & L;
  const uint32_t eq = ~(a1 ^ b1) & L;
  const uint32_t lo = (eq & (a0 | b0)) | (a1 & ~b1 & a0) | (b1 & ~a1 & b0);
  return ((a1 | b1) << 1) | lo;
}

// One thread per output word (b in {2, 4, 8}) or 32-code chunk (b = 3).
__global__ void maxpool_kernel(ActView in, int k, int stride, int pad, ActView out, int units) {
  const int64_t rows = (int64_t)out.n * out.h * out.w * out.groups;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= rows * units) return;
  const int64_t r = t / units;
  const int wi = (int)(t % units);
  const int g = (int)(r % out.groups);
  const int64_t p = r / out.groups;
  const int ox = (int)(p % out.w);
  const int oy = (int)((p / out.w) % out.h);
  const int n = (int)(p / ((int64_t)out.w * out.h));
  uint32_t *dst = (uint32_t *)row_at(out, r);
  if (in.bits == 2) {
    uint32_t m = 0;
    for (int ky = 0; ky < k; ++ky) {
      const int iy = oy * stride - pad + ky;
      if (iy < 0 || iy >= in.h) continue;
      for (int kx = 0; kx < k; ++kx) {
        const int ix = ox * stride - pad + kx;
        if (ix < 0 || ix >= in.w) continue;
        const uint32_t *row = (const uint32_t *)(in.data + (((int64_t)n * in.h + iy) * in.w + ix) * in.pixel +
                                                 (int64_t)g * in.gstride);
        m = max2x16(m, row[wi]);
      }
    }
    const int used = out.cpg * 2 - wi * 32;  // code bits of this word inside the row
    dst[wi] = used >= 32 ? m : (m & ((1u << used) - 1u));
    return;
  }
  const int per = in.bits == 3 ? 32 : 32 / store_bits(in.bits);
  const int j0 = wi * per;
  const int nc = min(per, out.cpg - j0);
  int c[32];
  for (int j = 0; j < 32; ++j) c[j] = 0;  // codes are >= 0
  for (int ky = 0; ky < k; ++ky) {
    const int iy = oy * stride - pad + ky;
    if (iy < 0 || iy >= in.h) continue;
    for (int kx = 0; kx < k; ++kx) {
      const int ix = ox * stride - pad + kx;
      if (ix < 0 || ix >= in.w) continue;
      const uint8_t *row = in.data + (((int64_t)n * in.h + iy) * in.w + ix) * in.pixel + g * in.gstride;
      for (int j = 0; j < nc; ++j) c[j] = max(c[j], read_code(row, j0 + j, in.bits, 0));
    }
  }
  if (in.bits == 3) {
    uint32_t words[3];
    pack_chunk(c, nc, 3, words);
    dst[3 * wi] = words[0];
    dst[3 * wi + 1] = words[1];
    dst[3 * wi + 2] = words[2];
  } else {
    uint32_t w = 0;
    for (int j = 0; j < nc; ++j) w |= (uint32_t)c[j] << (j * store_bits(in.bits));
    dst[wi] = w;
  }
}

// 2-bit codes, group rows of a multiple of 16 bytes: one thread per 16-byte
// piece of one output pixel's group row; grid (pieces of a pixel row, oy, n).
__global__ void maxpool2_kernel(ActView in, int k, int stride, int pad, ActView out) {
  const int qpr = (int)(out.row / 16);  // pieces per group row
  const int per_px = out.groups * qpr;
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= out.w * per_px) return;
  const int ox = t / per_px;
  const int rem = t - ox * per_px;
  const int g = rem / qpr, q = rem - g * qpr;
  const int oy = blockIdx.y, n = blockIdx.z;
  uint4 m = make_uint4(0, 0, 0, 0);
  const int y0 = oy * stride - pad, x0 = ox * stride - pad;
  const int ylo = max(0, y0), yhi = min(in.h, y0 + k), xlo = max(0, x0), xhi = min(in.w, x0 + k);
  for (int iy = ylo; iy < yhi; ++iy)
    for (int ix = xlo; ix < xhi; ++ix) {
      const uint4 v = *(const uint4 *)(in.data + (((int64_t)n * in.h + iy) * in.w + ix) * in.pixel +
                                       (int64_t)g * in.gstride + 16 * q);
      m.x = max2x16(m.x, v.x);
      m.y = max2x16(m.y, v.y);
      m.z = max2x16(m.z, v.z);
      m.w = max2x16(m.w, v.w);
    }
  *(uint4 *)(out.data + (((int64_t)n * out.h + oy) * out.w + ox) * out.pixel + (int64_t)g * out.gstride + 16 * q) = m;
}

// ------------------------------------------------------------ zero border
// out = in with a border of `pad` zero pixels on every side (whole pixels
// copied as 4-byte words).  One thread per output word.
__global__ void pad_pixels_kernel(ActView in, int pad, ActView out, int64_t words) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= words) return;
  const int wpp = (int)(out.pixel / 4);
  const int64_t px = t / wpp;
  const int wi = (int)(t - px * wpp);
  const int x = (int)(px % out.w);
  const int64_t r = px / out.w;
  const int y = (int)(r % out.h);
  const int n = (int)(r / out.h);
  const int iy = y - pad, ix = x - pad;
  uint32_t v = 0;
  if (iy >= 0 && iy < in.h && ix >= 0 && ix < in.w)
    v = ((const uint32_t *)(in.data + (((int64_t)n * in.h + iy) * in.w + ix) * in.pixel))[wi];
  ((uint32_t *)out.data)[t] = v;
}

// kPadRows output rows (image, padded row y) per workgroup: 32-bit words,
// zero outside the input rectangle; a thread loads its word of every row
// before it stores any (independent loads in flight, no per-word division).
constexpr int kPadRows = 8;
__global__ void pad_rows_kernel(ActView in, int pad, ActView out, int rows) {
  const int r0 = (int)blockIdx.x * kPadRows;
  const int wpp = (int)(out.pixel / 4);
  const int row_words = out.w * wpp;
  const int lo = pad * wpp, hi = (pad + in.w) * wpp;
  for (int w = threadIdx.x; w < row_words; w += blockDim.x) {
    uint32_t v[kPadRows];
#pragma unroll
    for (int j = 0; j < kPadRows; ++j) {
      const int r = r0 + j;
      const int y = r % out.h, n = r / out.h, iy = y - pad;
      v[j] = 0u;
      if (r < rows && iy >= 0 && iy < in.h && w >= lo && w < hi)
        v[j] = ((const uint32_t *)(in.data + ((int64_t)n * in.h + iy) * in.w * in.pixel))[w - lo];
    }
#pragma unroll
    for (int j = 0; j < kPadRows; ++j)
      if (r0 + j < rows) ((uint32_t *)(out.data + (int64_t)(r0 + j) * out.w * out.pixel))[w] = v[j];
  }
}

// ------------------------------------------------------------ global sum
// 2-bit codes, at most 85 pixels (85 x 3 < 256), 16 | cpg: one thread per
// (image, group, word of 16 codes).  The word's codes k, k+4, k+8, k+12 sit
// in the four bytes of (w >> 2k) & 0x03030303, so four byte-lane
// accumulators sum all 16 codes without carries.
__global__ void avgsum2_kernel(ActView in, int32_t *out) {
  const int wpr = in.cpg / 16;  // words per group row
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= (int64_t)in.n * in.groups * wpr) return;
  const int wi = (int)(t % wpr);
  const int64_t r = t / wpr;
  const int g = (int)(r % in.groups);
  const int n = (int)(r / in.groups);
  const int hw = in.h * in.w;
  const uint8_t *base = in.data + (int64_t)n * hw * in.pixel + (int64_t)g * in.gstride + 4 * wi;
  uint32_t acc[4] = {0, 0, 0, 0};
  for (int p = 0; p < hw; ++p) {
    const uint32_t w = *(const uint32_t *)(base + (int64_t)p * in.pixel);
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) acc[kk] += (w >> (2 * kk)) & 0x03030303u;
  }
  int32_t *o = out + (int64_t)n * in.groups * in.cpg + (int64_t)g * in.cpg + 16 * wi;
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    const int4 v = make_int4((int)((acc[0] >> (8 * b)) & 255u), (int)((acc[1] >> (8 * b)) & 255u),
                             (int)((acc[2] >> (8 * b)) & 255u), (int)((acc[3] >> (8 * b)) & 255u));
    *(int4 *)(o + 4 * b) = v;
  }
}

// Same sums with one workgroup per (image, group) when 256 is a multiple of
// the words per row: thread (word, r) takes pixels r, r + R, ... (R = 256 /
// words), and the R partial byte-lane sums of a word are added in LDS.
// planes (nullable): also the FC's signed base-256 digit planes of the sums
// (P planes of count bytes), and logits row n zeroed for the FC's atomics.
__global__ __launch_bounds__(256) void avgsum2_wg_kernel(ActView in, int32_t *out, int8_t *planes, int P,
                                                        int64_t count, int32_t *logits, int cout) {
  __shared__ uint32_t part[4][256];
  const int wpr = in.cpg / 16;
  const int R = 256 / wpr;
  const int n = (int)(blockIdx.x / in.groups), g = (int)(blockIdx.x % in.groups);
  const int wi = threadIdx.x % wpr, r = threadIdx.x / wpr;
  const int hw = in.h * in.w;
  const uint8_t *base = in.data + (int64_t)n * hw * in.pixel + (int64_t)g * in.gstride + 4 * wi;
  uint32_t acc[4] = {0, 0, 0, 0};
  // eight pixels' loads in flight before their sums
  for (int p0 = r; p0 < hw; p0 += 8 * R) {
    uint32_t w[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int p = p0 + u * R;
      w[u] = p < hw ? *(const uint32_t *)(base + (int64_t)p * in.pixel) : 0u;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u)
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) acc[kk] += (w[u] >> (2 * kk)) & 0x03030303u;
  }
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) part[kk][threadIdx.x] = acc[kk];
  __syncthreads();
  for (int idx = threadIdx.x; idx < 4 * wpr; idx += 256) {
    const int w2 = idx >> 2, kk = idx & 3;
    uint32_t sum = 0;
    for (int rr = 0; rr < R; ++rr) sum += part[kk][rr * wpr + w2];
    const int64_t c0 = (int64_t)n * in.groups * in.cpg + (int64_t)g * in.cpg + 16 * w2 + kk;
    int32_t *o = out + c0;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int32_t v = (int32_t)((sum >> (8 * b)) & 255u);
      o[4 * b] = v;
      if (planes) {  // v <= 255: digits v (one plane, v <= 127) or v - 256 and 1
        const int d0 = (int)(int8_t)(uint8_t)v;
        planes[c0 + 4 * b] = (int8_t)d0;
        if (P > 1) planes[count + c0 + 4 * b] = (int8_t)((v - d0) >> 8);
        for (int p = 2; p < P; ++p) planes[p * count + c0 + 4 * b] = 0;
      }
    }
  }
  if (logits && g == 0)
    for (int i = threadIdx.x; i < cout; i += 256) logits[(int64_t)n * cout + i] = 0;
}
__global__ void avgsum_kernel(ActView in, int32_t *out) {
  const int64_t C = (int64_t)in.groups * in.cpg;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= (int64_t)in.n * C) return;
  const int n = (int)(t / C);
  const int c = (int)(t % C);
  const int g = c / in.cpg, j = c % in.cpg;
  int32_t s = 0;
  const int64_t hw = (int64_t)in.h * in.w;
  for (int64_t p = 0; p < hw; ++p)
    s += read_code(in.data + ((int64_t)n * hw + p) * in.pixel + g * in.gstride, j, in.bits, 0);
  out[t] = s;
}

// ------------------------------------------------------------ FC
// Workgroup tile: 64 images x 64 outputs over a K slice of FC_KS features,
// staged through LDS; each thread owns a 4 x 4 block of outputs.  K slices
// are summed with integer atomics (order-free, hence exact).
constexpr int FC_T = 64, FC_KC = 64, FC_KS = 256;

__global__ void fill_i32_kernel(int32_t *p, int64_t n) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t < n) p[t] = 0;
}

__global__ __launch_bounds__(256) void fc_kernel(const int32_t *x, int n, int cin, const int8_t *w,
                                                 int cout, int32_t *logits) {
  __shared__ int32_t xs[FC_KC][FC_T + 1];
  __shared__ int32_t ws[FC_KC][FC_T + 1];
  const int i0 = blockIdx.y * FC_T, o0 = blockIdx.x * FC_T;
  const int c_begin = blockIdx.z * FC_KS;
  const int c_end = min(cin, c_begin + FC_KS);
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;  // outputs o0+4tx.., images i0+4ty..
  uint32_t acc[4][4];
  for (int a = 0; a < 4; ++a)
    for (int b = 0; b < 4; ++b) acc[a][b] = 0;
  for (int c0 = c_begin; c0 < c_end; c0 += FC_KC) {
    for (int e = threadIdx.x; e < FC_KC * FC_T; e += 256) {
      const int cc = e % FC_KC, rr = e / FC_KC;
      const int c = c0 + cc;
      const bool cok = c < c_end;
      xs[cc][rr] = (cok && i0 + rr < n) ? x[(int64_t)(i0 + rr) * cin + c] : 0;
      ws[cc][rr] = (cok && o0 + rr < cout) ? (int32_t)w[(int64_t)(o0 + rr) * cin + c] : 0;
    }
    __syncthreads();
    for (int cc = 0; cc < FC_KC; ++cc) {
      uint32_t xv[4], wv[4];
      for (int a = 0; a < 4; ++a) xv[a] = (uint32_t)xs[cc][4 * ty + a];
      for (int b = 0; b < 4; ++b) wv[b] = (uint32_t)ws[cc][4 * tx + b];
      for (int a = 0; a < 4; ++a)
        for (int b = 0; b < 4; ++b) acc[a][b] += xv[a] * wv[b];  // modular int32
    }
    __syncthreads();
  }
  for (int a = 0; a < 4; ++a) {
    const int i = i0 + 4 * ty + a;
    if (i >= n) continue;
    for (int b = 0; b < 4; ++b) {
      const int o = o0 + 4 * tx + b;
      if (o < cout) atomicAdd((uint32_t *)&logits[(int64_t)i * cout + o], acc[a][b]);
    }
  }
}

// FC on the matrix cores.  x = d0 + d1 256 + d2 256^2 + d3 256^3 (mod 2^32)
// with signed digits d_p in [-128, 127] (each taken from what remains after
// the lower ones, so the sum is exact modulo 2^32), so
// logits = sum_p 256^p (D_p W^T) with four int8 x int8 -> int32 products,
// each exact modulo 2^32 like the definition.  Digit planes: int8
// [4][n][cin].

// Four consecutive features per thread (cin % 16 == 0); also clears the
// logits, which fc_mfma_kernel's K slices add into.
template <int P>
__global__ void fc_digits_kernel(const int32_t *x, int64_t count, int8_t *planes, int32_t *logits,
                                 int64_t nlogits) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (int64_t i = t; i < nlogits; i += (int64_t)gridDim.x * blockDim.x) logits[i] = 0;
  if (4 * t >= count) return;
  const int4 v4 = *(const int4 *)(x + 4 * t);
  const int32_t v[4] = {v4.x, v4.y, v4.z, v4.w};
  uint32_t word[P] = {};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    int64_t r = v[e];
#pragma unroll
    for (int p = 0; p < P; ++p) {
      const int d = (int)(int8_t)(uint8_t)(r & 255);  // signed digit
      word[p] |= (uint32_t)(uint8_t)d << (8 * e);
      r = (r - d) >> 8;                                 // exact: r - d is a multiple of 256
    }
  }
#pragma unroll
  for (int p = 0; p < P; ++p) *(uint32_t *)(planes + p * count + 4 * t) = word[p];
}

typedef int v4i_t __attribute__((ext_vector_type(4)));
typedef int v16i_t __attribute__((ext_vector_type(16)));

// Workgroup: 32 outputs x 32 images x one K slice (blockIdx.z of
// gridDim.z); its 4 waves take every 4th 32-wide K step of the slice, sum
// their partial blocks in LDS and add the result to the logits (integer
// atomics: order-free, exact modulo 2^32).  A = weights (rows = outputs),
// B = one digit plane (columns = images); rows and images past the end
// read out-of-range offsets (zeros).
template <int P>
__global__ __launch_bounds__(256) void fc_mfma_kernel(const int8_t *w, const int8_t *planes, int n, int cin,
                                                      int cout, int32_t *logits) {
  __shared__ int32_t part[3][16][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int l32 = lane & 31, half = lane >> 5;
  const int o0 = blockIdx.x * 32, i0 = blockIdx.y * 32;
  const int64_t plane = (int64_t)n * cin;
  const auto rw = __builtin_amdgcn_make_buffer_rsrc((void *)w, (short)0, (int)((int64_t)cout * cin), 0x00020000);
  const auto rd = __builtin_amdgcn_make_buffer_rsrc((void *)planes, (short)0, (int)(P * plane), 0x00020000);
  const uint32_t kOut = 0x80000000u;  // past every buffer this kernel reads
  const uint32_t wrow = o0 + l32 < cout ? (uint32_t)((o0 + l32) * cin + 16 * half) : kOut;
  const uint32_t drow = i0 + l32 < n ? (uint32_t)((i0 + l32) * cin + 16 * half) : kOut;
  v16i_t acc[P];
#pragma unroll
  for (int p = 0; p < P; ++p)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[p][r] = 0;
  const int steps = cin / 32;
  const int per = (steps + gridDim.z - 1) / gridDim.z;
  const int k_end = 32 * min(steps, per * (int)(blockIdx.z + 1));
  // the wave's K steps k, k + 128, ...: the operands of U steps are loaded
  // before their MFMAs, so that U loads are in flight at once
  constexpr int U = 4;
  auto wload = [&](int k) __attribute__((always_inline)) {
    return __builtin_bit_cast(v4i_t, __builtin_amdgcn_raw_buffer_load_b128(rw, (int)(wrow + k), 0, 0));
  };
  auto dload = [&](int k, int p) __attribute__((always_inline)) {
    const uint32_t off = drow == kOut ? kOut : drow + (uint32_t)(p * plane) + k;
    return __builtin_bit_cast(v4i_t, __builtin_amdgcn_raw_buffer_load_b128(rd, (int)off, 0, 0));
  };
  int k = 32 * (per * (int)blockIdx.z + wave);
  for (; k + 128 * (U - 1) < k_end; k += 128 * U) {
    v4i_t a[U], b[U][P];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      a[u] = wload(k + 128 * u);
#pragma unroll
      for (int p = 0; p < P; ++p) b[u][p] = dload(k + 128 * u, p);
    }
    __builtin_amdgcn_sched_barrier(0);  // every load issued before the first wait
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int p = 0; p < P; ++p) acc[p] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[u], b[u][p], acc[p], 0, 0, 0);
  }
  for (; k < k_end; k += 128) {
    const v4i_t a = wload(k);
#pragma unroll
    for (int p = 0; p < P; ++p) acc[p] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, dload(k, p), acc[p], 0, 0, 0);
  }
  uint32_t tot[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    tot[r] = 0;
#pragma unroll
    for (int p = 0; p < P; ++p) tot[r] += (uint32_t)acc[p][r] << (8 * p);
  }
  if (wave > 0)
#pragma unroll
    for (int r = 0; r < 16; ++r) part[wave - 1][r][lane] = (int32_t)tot[r];
  __syncthreads();
  if (wave != 0) return;
  const int i = i0 + l32;
  if (i >= n) return;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int o = o0 + 8 * (r >> 2) + 4 * half + (r & 3);
    const uint32_t sum = tot[r] + (uint32_t)part[0][r][lane] + (uint32_t)part[1][r][lane] + (uint32_t)part[2][r][lane];
    if (o < cout) atomicAdd((uint32_t *)&logits[(int64_t)i * cout + o], sum);
  }
}

}  // namespace

size_t fc_scratch_bytes(int n, int cin) { return cin % 32 == 0 ? (size_t)4 * n * cin : 0; }

hipError_t launch_pack(const void *codes, const ActView &out, hipStream_t s) {
  const int64_t rows = (int64_t)out.n * out.h * out.w * out.groups;
  const int chunks = (out.cpg + 31) / 32;
  if (rows == 0) return hipSuccess;
  hipLaunchKernelGGL(pack_kernel, dim3(grid_for(rows * chunks)), dim3(kBlock), 0, s,
                     (const uint8_t *)codes, out, rows, chunks);
  return hipGetLastError();
}

hipError_t launch_unpack(const ActView &in, void *codes, hipStream_t s) {
  const int64_t rows = (int64_t)in.n * in.h * in.w * in.groups;
  const int chunks = (in.cpg + 31) / 32;
  if (rows == 0) return hipSuccess;
  hipLaunchKernelGGL(unpack_kernel, dim3(grid_for(rows * chunks)), dim3(kBlock), 0, s, in,
                     (uint8_t *)codes, rows, chunks);
  return hipGetLastError();
}

hipError_t launch_minmax(const float *x, int64_t count, float *range, hipStream_t s) {
  uint32_t *enc = (uint32_t *)range;
  hipLaunchKernelGGL(range_init_kernel, dim3(1), dim3(1), 0, s, enc);
  if (count > 0) {
    int64_t g = (count + kBlock - 1) / kBlock;
    if (g > 4096) g = 4096;
    hipLaunchKernelGGL(minmax_kernel, dim3((unsigned)g), dim3(kBlock), 0, s, x, count, enc);
  }
  return hipGetLastError();
}

// Four 3-channel 8-bit pixels per thread with 16-byte loads and stores.
bool quantize_by_pixels(const float *x, const ActView &out) {
  const int64_t rows = (int64_t)out.n * out.h * out.w * out.groups;
  return out.bits == 8 && out.cpg == 3 && out.groups == 1 && out.row == 4 && rows % 4 == 0 &&
         (((uintptr_t)x | (uintptr_t)out.data) & 15u) == 0;
}

const char *quantize_label(const float *x, const ActView &out) {
  return quantize_by_pixels(x, out) ? "quantize_px3_kernel" : "quantize_kernel";
}

hipError_t launch_quantize(const float *x, float l, float u, const float *range, const ActView &out,
                           hipStream_t s) {
  const int64_t rows = (int64_t)out.n * out.h * out.w * out.groups;
  const int units = out.bits == 3 ? (out.cpg + 31) / 32 : (int)(out.row / 4);
  if (rows == 0) return hipSuccess;
  if (quantize_by_pixels(x, out)) {
    hipLaunchKernelGGL(quantize_px3_kernel, dim3(grid_for(rows / 4)), dim3(kBlock), 0, s, x, l, u,
                       (const uint32_t *)range, out, rows / 4);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(quantize_kernel, dim3(grid_for(rows * units)), dim3(kBlock), 0, s, x, l, u,
                     (const uint32_t *)range, out, rows, units);
  return hipGetLastError();
}

// Four input pixels per thread with 16-byte loads (rows of up to 256 + 2 pad
// pixels, 4-byte output pixels, 16-byte aligned input).
bool quantize_pad_vector(const float *x, int in_w, int pad, const ActView &out) {
  return in_w % 4 == 0 && in_w / 4 + 2 * pad <= 64 && out.pixel == 4 && ((uintptr_t)x & 15u) == 0;
}

const char *quantize_pad_label(const float *x, int in_w, int pad, const ActView &out) {
  return quantize_pad_vector(x, in_w, pad, out) ? "quantize_pad4_kernel" : "quantize_pad_kernel";
}

hipError_t launch_quantize_pad(const float *x, float l, float u, int in_h, int in_w, int pad, const ActView &out,
                               hipStream_t s) {
  const int64_t rows = (int64_t)out.n * out.h;
  if (rows == 0 || out.w == 0) return hipSuccess;
  if (rows >= 0x7fffffff) return hipErrorInvalidValue;
  if (quantize_pad_vector(x, in_w, pad, out)) {
    hipLaunchKernelGGL(quantize_pad4_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s, x, l, u, in_h, in_w,
                       pad, out, (int)rows);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(quantize_pad_kernel, dim3((unsigned)((rows + kQPadRows - 1) / kQPadRows)), dim3(256), 0, s, x,
                     l, u, in_h, in_w, pad, out, (int)rows);
  return hipGetLastError();
}

hipError_t launch_range_out(const float *enc, float *range_out, hipStream_t s) {
  hipLaunchKernelGGL(range_out_kernel, dim3(1), dim3(1), 0, s, (const uint32_t *)enc, range_out);
  return hipGetLastError();
}

hipError_t launch_shuffle(const ActView &in, int32_t steps, const ActView &out, hipStream_t s) {
  const int64_t pixels = (int64_t)in.n * in.h * in.w;
  const int64_t items = pixels * in.groups * (in.row / 4);
  if (items == 0) return hipSuccess;
  hipLaunchKernelGGL(shuffle_kernel, dim3(grid_for(items)), dim3(kBlock), 0, s, in, steps, out,
                     pixels);
  return hipGetLastError();
}

// The word-level build: b in {2, 4, 8}, rows without padding (C a multiple
// of the codes per word), a pixel a whole number of 16-byte stores (in the
// group layout, each row), G a power of two up to 16 and both tensors
// 16-byte aligned.
static bool channel_shuffle_words(const ActView &in, const ActView &out) {
  const int b = in.bits, G = in.groups;
  if (b != 2 && b != 4 && b != 8) return false;
  if (G != 2 && G != 4 && G != 8 && G != 16) return false;
  const int F = 32 / b;
  // a pixel's output rows are one run in the pixel layout; in the group
  // layout every 16-byte store must stay inside one row
  const bool run = out.gstride == out.row;
  return in.cpg % F == 0 && ((int64_t)G * in.cpg) % (4 * F) == 0 && (run || out.row % 16 == 0) &&
         (((uintptr_t)in.data | (uintptr_t)out.data) & 15u) == 0 &&
         (int64_t)G * in.cpg / (4 * F) < ((int64_t)1 << 30);
}

const char *channel_shuffle_label(const ActView &in, const ActView &out) {
  return channel_shuffle_words(in, out) ? "channel_shuffle_words_kernel" : "channel_shuffle_kernel";
}

template <int B>
static hipError_t launch_channel_shuffle_words(const ActView &in, const ActView &out, int64_t threads, int tpp,
                                        hipStream_t s) {
  switch (in.groups) {
    case 2: hipLaunchKernelGGL((channel_shuffle_words_kernel<B, 2>), dim3(grid_for(threads)), dim3(kBlock), 0, s, in, out, threads, tpp); break;
    case 4: hipLaunchKernelGGL((channel_shuffle_words_kernel<B, 4>), dim3(grid_for(threads)), dim3(kBlock), 0, s, in, out, threads, tpp); break;
    case 8: hipLaunchKernelGGL((channel_shuffle_words_kernel<B, 8>), dim3(grid_for(threads)), dim3(kBlock), 0, s, in, out, threads, tpp); break;
    default: hipLaunchKernelGGL((channel_shuffle_words_kernel<B, 16>), dim3(grid_for(threads)), dim3(kBlock), 0, s, in, out, threads, tpp); break;
  }
  return hipGetLastError();
}

hipError_t launch_channel_shuffle(const ActView &in, const ActView &out, hipStream_t s) {
  const int64_t pixels = (int64_t)in.n * in.h * in.w;
  if (pixels > 0 && channel_shuffle_words(in, out)) {
    const int tpp = (int)(in.row * in.groups / 16);
    const int64_t threads = pixels * tpp;
    if (in.bits == 2) return launch_channel_shuffle_words<2>(in, out, threads, tpp, s);
    if (in.bits == 4) return launch_channel_shuffle_words<4>(in, out, threads, tpp, s);
    return launch_channel_shuffle_words<8>(in, out, threads, tpp, s);
  }
  const int chunks = (in.cpg + 31) / 32;
  const int64_t items = pixels * in.groups * chunks;
  if (items == 0) return hipSuccess;
  hipLaunchKernelGGL(channel_shuffle_kernel, dim3(grid_for(items)), dim3(kBlock), 0, s, in, out, pixels,
                     chunks);
  return hipGetLastError();
}

// 2-bit rows of a multiple of 16 bytes: 64 codes per thread (SWAR max).
bool maxpool_vector(const ActView &in, const ActView &out) {
  return in.bits == 2 && out.row % 16 == 0 && out.h <= 65535 && out.n <= 65535 &&
         (((uintptr_t)in.data | (uintptr_t)out.data) & 15u) == 0 &&
         (int64_t)out.w * out.groups * (out.row / 16) < ((int64_t)1 << 30);
}

const char *maxpool_label(const ActView &in, const ActView &out) {
  return maxpool_vector(in, out) ? "maxpool2_kernel" : "maxpool_kernel";
}

hipError_t launch_maxpool(const ActView &in, int k, int stride, int pad, const ActView &out,
                          hipStream_t s) {
  const int64_t rows = (int64_t)out.n * out.h * out.w * out.groups;
  const int units = out.bits == 3 ? (out.cpg + 31) / 32 : (int)(out.row / 4);
  if (rows == 0) return hipSuccess;
  if (maxpool_vector(in, out)) {
    const int64_t per_row = (int64_t)out.w * out.groups * (out.row / 16);
    dim3 grid((unsigned)((per_row + kBlock - 1) / kBlock), (unsigned)out.h, (unsigned)out.n);
    hipLaunchKernelGGL(maxpool2_kernel, grid, dim3(kBlock), 0, s, in, k, stride, pad, out);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(maxpool_kernel, dim3(grid_for(rows * units)), dim3(kBlock), 0, s, in, k,
                     stride, pad, out, units);
  return hipGetLastError();
}

bool pad_by_rows(const ActView &out) {
  return (int64_t)out.n * out.h < 0x7fffffff && (int64_t)out.w * out.pixel < 0x7fffffff;
}

const char *pad_pixels_label(const ActView &out) { return pad_by_rows(out) ? "pad_rows_kernel" : "pad_pixels_kernel"; }

hipError_t launch_pad_pixels(const ActView &in, int pad, const ActView &out, hipStream_t s) {
  const int64_t words = (int64_t)out.n * out.h * out.w * (out.pixel / 4);
  if (words == 0) return hipSuccess;
  const int64_t rows = (int64_t)out.n * out.h;
  if (pad_by_rows(out)) {
    hipLaunchKernelGGL(pad_rows_kernel, dim3((unsigned)((rows + kPadRows - 1) / kPadRows)), dim3(256), 0, s, in, pad,
                       out, (int)rows);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(pad_pixels_kernel, dim3(grid_for(words)), dim3(kBlock), 0, s, in, pad, out, words);
  return hipGetLastError();
}

bool avgsum_makes_fc_planes(const ActView &in) {
  const int wpr = in.cpg / 16;
  return in.bits == 2 && in.cpg % 16 == 0 && (int64_t)in.h * in.w <= 85 && wpr >= 1 && wpr <= 256 &&
         256 % wpr == 0 && (int64_t)in.n * in.groups < ((int64_t)1 << 31);
}

int fc_planes(int64_t xmax) { return xmax >= 0 && xmax <= 127 ? 1 : xmax >= 0 && xmax <= 32639 ? 2 : 4; }

// 0: one thread per channel; 1: byte-lane sums of 2-bit rows (16 codes per
// thread); 2: the same with one workgroup per image row block (which can
// also write the FC's digit planes).
int avgsum_path(const ActView &in, const int32_t *out) {
  if (in.bits == 2 && in.cpg % 16 == 0 && (int64_t)in.h * in.w <= 85) {
    const int wpr = in.cpg / 16;
    if (wpr <= 256 && 256 % wpr == 0 && (int64_t)in.n * in.groups < ((int64_t)1 << 31)) return 2;
    if (((uintptr_t)out & 15u) == 0) return 1;
  }
  return 0;
}

const char *avgsum_label(const ActView &in, const int32_t *out) {
  static const char *names[3] = {"avgsum_kernel", "avgsum2_kernel", "avgsum2_wg_kernel"};
  return names[avgsum_path(in, out)];
}

hipError_t launch_avgsum(const ActView &in, int32_t *out, hipStream_t s, int8_t *planes, int P, int32_t *logits,
                         int cout) {
  const int64_t items = (int64_t)in.n * in.groups * in.cpg;
  if (items == 0) return hipSuccess;
  if (planes && !avgsum_makes_fc_planes(in)) return hipErrorInvalidValue;
  const int path = avgsum_path(in, out);
  if (path == 2) {
    hipLaunchKernelGGL(avgsum2_wg_kernel, dim3((unsigned)(in.n * in.groups)), dim3(256), 0, s, in, out, planes, P,
                       items, logits, cout);
    return hipGetLastError();
  }
  if (path == 1) {
    hipLaunchKernelGGL(avgsum2_kernel, dim3(grid_for(items / 16)), dim3(kBlock), 0, s, in, out);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(avgsum_kernel, dim3(grid_for(items)), dim3(kBlock), 0, s, in, out);
  return hipGetLastError();
}

bool fc_mfma_applies(const int32_t *x, int n, int cin, int cout, const int8_t *scratch) {
  return scratch && cin % 32 == 0 && ((uintptr_t)x & 15u) == 0 && (int64_t)4 * n * cin < ((int64_t)1 << 31) &&
         (int64_t)cout * cin < ((int64_t)1 << 31);
}

const char *fc_label(const int32_t *x, int n, int cin, int cout, const int8_t *scratch, bool planes_ready) {
  if (!fc_mfma_applies(x, n, cin, cout, scratch)) return "fill_i32_kernel + fc_kernel";
  return planes_ready ? "fc_mfma_kernel" : "fc_digits_kernel + fc_mfma_kernel";
}

hipError_t launch_fc(const int32_t *x, int n, int cin, const int8_t *w, int cout, int32_t *logits,
                     int8_t *scratch, hipStream_t s, int64_t xmax, bool planes_ready) {
  const int64_t items = (int64_t)n * cout;
  if (items == 0) return hipSuccess;
  if (fc_mfma_applies(x, n, cin, cout, scratch)) {
    const int64_t count = (int64_t)n * cin;
    // signed base-256 digit planes: one covers |x| <= 127, two |x| <= 32639,
    // four every int32 (exact modulo 2^32); planes_ready: the global sum
    // wrote them and zeroed the logits
    const int P = fc_planes(xmax);
    if (!planes_ready) {
      auto digits = P == 1 ? fc_digits_kernel<1> : P == 2 ? fc_digits_kernel<2> : fc_digits_kernel<4>;
      hipLaunchKernelGGL(digits, dim3(grid_for(count / 4)), dim3(kBlock), 0, s, x, count, scratch, logits, items);
    }
    // K slices (of at least 4 steps) for about 128 workgroups: more slices
    // only add contended atomics (ResNet-18 batch 64: 2 slices 16 us, 8
    // slices 20 us, 32 slices 48 us)
    const int64_t blocks = (int64_t)((cout + 31) / 32) * ((n + 31) / 32);
    int slices = (int)std::max<int64_t>(1, std::min<int64_t>((128 + blocks - 1) / blocks, cin / 128));
    dim3 grid((unsigned)((cout + 31) / 32), (unsigned)((n + 31) / 32), (unsigned)slices);
    auto mm = P == 1 ? fc_mfma_kernel<1> : P == 2 ? fc_mfma_kernel<2> : fc_mfma_kernel<4>;
    hipLaunchKernelGGL(mm, grid, dim3(256), 0, s, w, (const int8_t *)scratch, n, cin, cout, logits);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(fill_i32_kernel, dim3(grid_for(items)), dim3(kBlock), 0, s, logits, items);
  dim3 grid((unsigned)((cout + FC_T - 1) / FC_T), (unsigned)((n + FC_T - 1) / FC_T),
            (unsigned)((cin + FC_KS - 1) / FC_KS));
  hipLaunchKernelGGL(fc_kernel, grid, dim3(256), 0, s, x, n, cin, w, cout, logits);
  return hipGetLastError();
}

}  // namespace palq
