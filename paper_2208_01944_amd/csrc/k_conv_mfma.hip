// Grouped B-bit convolution as an implicit GEMM on gfx950 int8 MFMA.
//
// Per group g (Section 4.1: G independent B-bit convolutions) the layer is
// D[k][m] = sum_K W[k][K] X[K][m] (Eq. 1) with k an output channel of the
// group, m an output pixel (n, oy, ox) and K = (ky, kx, c), contracted with
// v_mfma_i32_32x32x32_i8: A = weights (rows = channels), B = activations
// (columns = pixels), int32 accumulation.
//
//  * Weights are prepacked once per layer (prepack_kernel): sign-extended to
//    int8, in MFMA operand order, 2 KB per (64-code K-block, 32 channels).
//    A persistent workgroup copies the whole K extent of its 32 or 64
//    channels into LDS once and keeps it there.
//  * Activations stay packed in HBM; each lane reads its own pixel's codes
//    for the current tap with a buffer load (out-of-image taps and pixels
//    past the end use an out-of-range offset, which the hardware returns as
//    zero) and unpacks them in registers with a few shift/mask operations.
//    The K order inside a 16-code unit is permuted by the unpack; the
//    weights are prepacked with the same permutation, which leaves the
//    contraction unchanged.
//  * 2-bit codes: the unpack leaves code 4e+d of a unit at bits 2d..2d+1 of
//    byte e without shifting it down (d = 0, 1, 2) or after one shift
//    (d = 3), i.e. scaled by 1, 4, 16, 16; the weights of those positions
//    are pre-scaled by 16, 4, 1, 1 so every product carries the factor 16,
//    which the epilogue removes exactly.
//  * Epilogue: accumulator + shortcut -> exact fixed-point requant with
//    ReLU -> b-bit codes, written to group (g + s) mod G: the cyclic
//    permutation of Eq. 8 is only the store address.  A projection shortcut
//    is fused as extra K-blocks (1x1 conv of the block input of the
//    destination group), so its accumulator lands in the same registers.
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <type_traits>

#include "codes.h"
#include "palq_internal.h"

namespace palq {

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef int v2i __attribute__((ext_vector_type(2)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef float v4f __attribute__((ext_vector_type(4)));


// ---------------------------------------------------------------- unpack
// Activation unit (16 unsigned codes) -> MFMA operand (16 int8), and the
// matching weight unit -> operand in the same K order.

// B = 2: one packed word per unit.
__device__ inline v4i act_unpack2(uint32_t x) {
  v4i r;
  r[0] = (int)(x & 0x03030303u);
  r[1] = (int)(x & 0x0C0C0C0Cu);
  r[2] = (int)(x & 0x30303030u);
  r[3] = (int)((x >> 2) & 0x30303030u);
  return r;
}
// Signed 2-bit weight unit -> int8 scaled by 16, 4, 1, 1 for d = 0..3.
__device__ inline v4i wt_unpack2(uint32_t y) {
  v4i r;
  // v_perm_b32 byte lookup: selector byte c in 0..3 picks byte c of the
  // table word, which holds sext(c) * scale.
  r[0] = (int)__builtin_amdgcn_perm(0u, 0xF0E01000u, y & 0x03030303u);          // x16
  r[1] = (int)__builtin_amdgcn_perm(0u, 0xFCF80400u, (y >> 2) & 0x03030303u);   // x4
  r[2] = (int)__builtin_amdgcn_perm(0u, 0xFFFE0100u, (y >> 4) & 0x03030303u);   // x1
  r[3] = (int)__builtin_amdgcn_perm(0u, 0xFFFE0100u, (y >> 6) & 0x03030303u);   // x1
  return r;
}

// B = 4: two packed words per unit; byte (d, e) = code 8*(d>>1) + 2e + (d&1).
__device__ inline v4i unpack4_nibbles(uint32_t y0, uint32_t y1) {
  v4i r;
  r[0] = (int)(y0 & 0x0F0F0F0Fu);
  r[1] = (int)((y0 >> 4) & 0x0F0F0F0Fu);
  r[2] = (int)(y1 & 0x0F0F0F0Fu);
  r[3] = (int)((y1 >> 4) & 0x0F0F0F0Fu);
  return r;
}
// Per-byte sign extension of b-bit fields (values 0 .. 2^b - 1 in each byte):
// ((v ^ s) + (0x80 - s)) ^ 0x80 with s = 2^(b-1) never carries across bytes.
template <int B>
__device__ inline uint32_t sext_bytes(uint32_t v) {
  constexpr uint32_t s = 0x01010101u << (B - 1);
  constexpr uint32_t k = 0x80808080u - s;
  return ((v ^ s) + k) ^ 0x80808080u;
}
__device__ inline v4i wt_unpack4(uint32_t y0, uint32_t y1) {
  v4i r = unpack4_nibbles(y0, y1);
  _Pragma("unroll") for (int d = 0; d < 4; ++d) r[d] = (int)sext_bytes<4>((uint32_t)r[d]);
  return r;
}

// B = 3: unit j (0/1) of a 32-code chunk: low word lo = bits 0-1 of its 16
// codes, hi = the chunk's bit-2 word (bit 8e + 2d + j for code 4e + d of
// unit j).
__device__ inline v4i unpack3(uint32_t lo, uint32_t hi, int j) {
  v4i r;
  _Pragma("unroll") for (int d = 0; d < 4; ++d) {
    const uint32_t l2 = (lo >> (2 * d)) & 0x03030303u;
    const uint32_t h1 = (hi >> (2 * d + j)) & 0x01010101u;
    r[d] = (int)(l2 | (h1 << 2));
  }
  return r;
}
__device__ inline v4i wt_unpack3(uint32_t lo, uint32_t hi, int j) {
  v4i r = unpack3(lo, hi, j);
  _Pragma("unroll") for (int d = 0; d < 4; ++d) r[d] = (int)sext_bytes<3>((uint32_t)r[d]);
  return r;
}

// Bytes of packed data per 64-code K-block row and per lane (half a block).
template <int B> struct Blk {
  static constexpr int bytes = 8 * B;       // 64 codes
  static constexpr int lane_words = B;      // 32 codes = B words (3 for B = 3)
};

// Raw packed words a lane holds for one K-block (its half: two units); the
// stem layout holds eight 4-byte pixels.
template <int B, bool STEM> struct RawT { uint32_t w[STEM ? 8 : B]; };

// MFMA B operand for K-step j (0/1) from a lane's raw half block.  B = 8
// (unsigned 8-bit codes, and 6-bit codes stored one per byte): the bytes
// with their top bit flipped, x - 128 as int8; the kernel starts each
// accumulator at 128 sum(w) of its channel (Geo::acc0), which restores
// sum(w x) exactly, out-of-image taps included (their code 0 reads as -128
// as well).
template <int B>
__device__ inline v4i act_operand(const RawT<B, false> &r, int j) {
  if constexpr (B == 2) return act_unpack2(r.w[j]);
  else if constexpr (B == 4) return unpack4_nibbles(r.w[2 * j], r.w[2 * j + 1]);
  else if constexpr (B == 8)
    return v4i{(int)(r.w[4 * j] ^ 0x80808080u), (int)(r.w[4 * j + 1] ^ 0x80808080u),
               (int)(r.w[4 * j + 2] ^ 0x80808080u), (int)(r.w[4 * j + 3] ^ 0x80808080u)};
  else return unpack3(r.w[j], r.w[2], j);
}

// Weight unit u (0..3) of a 64-code K-block starting at p -> operand.
template <int B>
__device__ inline v4i load_weight_unit(const uint8_t *p, int u) {
  const uint32_t *q = (const uint32_t *)p;
  if constexpr (B == 2) return wt_unpack2(q[u]);
  else if constexpr (B == 4) return wt_unpack4(q[2 * u], q[2 * u + 1]);
  else if constexpr (B == 8) return v4i{(int)q[4 * u], (int)q[4 * u + 1], (int)q[4 * u + 2], (int)q[4 * u + 3]};
  else return wt_unpack3(q[3 * (u >> 1) + (u & 1)], q[3 * (u >> 1) + 2], u & 1);
}

// ---------------------------------------------------------------- requant
// Exact fixed-point requant with an int64 product (fallback path).
__device__ inline int requant_mul(int64_t t, int32_t m, int32_t sh, int qmax) {
  const int64_t num = t * (int64_t)m + ((int64_t)1 << (sh - 1));
  int64_t q = num >> sh;
  q = q < 0 ? 0 : q;
  return (int)(q > qmax ? qmax : q);
}

// Code j (0..31) of a 32-code chunk held in registers.
__device__ inline int chunk_code(const uint32_t *cw, int j, int bits) {
  if (bits == 3) {
    const uint32_t v = (cw[j >> 4] >> (2 * (j & 15))) & 3u;
    return (int)(v | (((cw[2] >> b3_hi_pos(j)) & 1u) << 2));
  }
  const int bit = j * store_bits(bits);
  return (int)((cw[bit >> 5] >> (bit & 31)) & ((1u << bits) - 1u));
}

// Codes of 4 consecutive channels c0..c0+3 (c0 % 4 == 0) of a packed row.
__device__ inline void row_quad(const uint8_t *row, int c0, int bits, int out[4]) {
  const uint32_t *w = (const uint32_t *)row;
  if (bits == 3) {
    const uint32_t *ch = w + 3 * (c0 >> 5);
    const int j0 = c0 & 31;
    const uint32_t lo = ch[j0 >> 4] >> (2 * (j0 & 15));
    const uint32_t hi = ch[2];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      out[e] = (int)(((lo >> (2 * e)) & 3u) | (((hi >> b3_hi_pos(j0 + e)) & 1u) << 2));
    return;
  }
  const int sb = store_bits(bits);
  const int bit = c0 * sb;
  const uint32_t v = w[bit >> 5] >> (bit & 31);
  const uint32_t mask = (1u << bits) - 1u;
#pragma unroll
  for (int e = 0; e < 4; ++e) out[e] = (int)((v >> (sb * e)) & mask);
}

// Per-channel requant constants in fp64.  With v = 2^lscale (acc + residual)
// (an integer, |v| < 2^31) and t = acc + residual + bias:
//   s = M 2^-(sh + lscale),  o = (bias M + 2^(sh-1)) 2^-sh,
//   fma(v, s, o) = (t M + 2^(sh-1)) 2^-sh exactly whenever |t| M < 2^52,
// so q = clamp(trunc(fma(v, s, o)), 0, qmax) equals the definition (trunc
// and floor differ only below zero, where both clamp to 0).  The prep kernel
// checks that bound for every channel from the accumulator bound; if any
// channel could break it, the layer's flag selects the int64 path instead.
struct RqConst {
  double s, o;
};

__global__ void requant_prep_kernel(const int32_t *mult, const int32_t *shift, const int32_t *bias,
                                    const int32_t *res_mult, int res_max, int nch, int lscale,
                                    int64_t acc_bound, RqConst *rq, int32_t *flag) {
  __shared__ int any;
  if (threadIdx.x == 0) any = 0;
  __syncthreads();
  int bad = 0;
  for (int c = threadIdx.x; c < nch; c += blockDim.x) {
    const int64_t m = mult[c];
    const int sh = shift[c];
    const int64_t b = bias ? bias[c] : 0;
    const int64_t rm = res_mult ? res_mult[c] : 0;
    RqConst k{0.0, 0.0};
    if (m < 0 || sh < 1 || sh > 62) {
      bad = 1;
    } else {
      const int64_t tmax = acc_bound + (b < 0 ? -b : b) + (rm < 0 ? -rm : rm) * res_max;
      const int64_t lim = (int64_t)1 << 52;
      if (m > 0 && tmax >= lim / m) bad = 1;
      const int64_t num = b * m + ((int64_t)1 << (sh - 1));  // |b m| < 2^61
      if (num >= lim || num <= -lim) bad = 1;
      k.s = ldexp((double)m, -sh - lscale);  // the accumulator is 2^lscale (acc + residual): exact
      k.o = ldexp((double)num, -sh);
    }
    rq[c] = k;
  }
  if (bad) atomicOr(&any, 1);
  __syncthreads();
  if (threadIdx.x == 0) *flag = any;
}

// The FP4 kernel's fp32 requant (2-bit outputs).  The accumulator starts at
// b4 = bias / 4 and adds the products as multiples of 1/4, so it holds
// u / 4 with u = t + bias (the identity shortcut's rm c / 4 added in fp32);
// every partial value is exact when |t| + |bias| + 3 |rm| < 2^24.  With
// sc = M 2^(2 - sh) (exact for |M| < 2^24) one fma gives
//   y = RN(u M 2^-sh + 1/2) = RN(x),  x = (u M + 2^(sh-1)) 2^-sh,
// a single rounding of x.  x 2^sh is an integer, so below an integer k <= 3
// x stays at least 2^-sh <= 2^-22 under k, more than half the fp32 spacing
// there (2^-23): RN(x) < k whenever x < k, and RN(x) >= floor(x) always.
// Hence min(trunc(y), 3) (v_cvt_u32_f32 truncates and takes negative values
// to 0) equals clamp(floor(x), 0, 3), the definition, for sh <= 22.  rm4:
// the shortcut scale res_mult / 4 (exact, |res_mult| < 2^15).  flag: 1 when
// every channel meets the bounds (else the fp64 epilogue runs).
__global__ void requant_prep_f32_kernel(const int32_t *mult, const int32_t *shift, const int32_t *bias,
                                        const int32_t *res_mult, int res_max, int nch, int64_t acc_bound, float *sc,
                                        float *b4, float *rm4, int32_t *flag) {
  __shared__ int any_bad;
  if (threadIdx.x == 0) any_bad = 0;
  __syncthreads();
  int bad = 0;
  for (int c = threadIdx.x; c < nch; c += blockDim.x) {
    const int64_t m = mult[c];
    const int sh = shift[c];
    const int64_t b = bias ? bias[c] : 0;
    const int64_t rm = res_mult ? res_mult[c] : 0;
    const int64_t lim = (int64_t)1 << 24;
    const int64_t umax = acc_bound + (b < 0 ? -b : b) + (rm < 0 ? -rm : rm) * res_max;
    if (sh < 1 || sh > 22 || m <= -lim || m >= lim || umax >= lim) bad = 1;
    sc[c] = bad ? 0.0f : ldexpf((float)m, 2 - sh);
    b4[c] = bad ? 0.0f : (float)b * 0.25f;
    rm4[c] = bad ? 0.0f : (float)rm * 0.25f;
  }
  if (bad) atomicOr(&any_bad, 1);
  __syncthreads();
  if (threadIdx.x == 0) *flag = any_bad ? 0 : 1;
}

// ---------------------------------------------------------------- geometry
struct Geo {
  int32_t M;          // output pixels per group
  int32_t cpb;        // 64-code K-blocks per tap (grouped mode)
  int32_t kb_main;    // K-blocks of the main convolution
  int32_t kb_total;   // + projection K-blocks
  int64_t w_ch;       // bytes of one output channel's filter
  int64_t pw_ch;      // bytes of one projection filter channel
  int32_t scale;      // operand scale of the accumulator (16 for 2-bit codes)
  const uint8_t *wp;  // weights in MFMA operand order (see prepack_kernel)
  const RqConst *rq;  // per-channel requant constants, then the int64-path flag
  const int32_t *acc0;  // B = 8: per-channel accumulator start 128 sum(w) (act_operand)
  float inv_hw, inv_wo;  // 1 / (ho wo) and 1 / wo, rounded to fp32 (fdiv's estimates)
};

// A (kb, 32-channel block) slab of prepacked weights: [j][half][ch][16 B].
constexpr int kSlab = 2048;
constexpr int kLdsBudget = 160 * 1024;  // gfx950 LDS per CU
constexpr int kNW = 8;                  // waves per workgroup

// Sign-extended (and, for 2-bit activations, scaled) weight unit u (0..3) of
// K-block kb for output channel k of group g: the 16 int8 values lane
// (ch, half = u >> 1) feeds to K-step j = u & 1.
template <int B, bool STEM>
__device__ inline v4i weight_unit(const ConvArgs &a, const Geo &geo, int g, int gd, int k, int kb, int u) {
  v4i v = {0, 0, 0, 0};
  if constexpr (STEM) {
    // unit u of K-block kb: filter row ky = 2 kb + (u >> 1), taps kx = 4 (u & 1) + d
    const int ky = 2 * kb + (u >> 1);
    if (ky < a.kh) {
      const uint32_t *wr = (const uint32_t *)(a.w + (((int64_t)g * a.cout + k) * a.kh + ky) * a.kw * 4);
      const uint32_t cmask = a.in.cpg >= 4 ? 0xffffffffu : ((1u << (8 * a.in.cpg)) - 1u);
#pragma unroll
      for (int d = 0; d < 4; ++d) {
        const int kx = 4 * (u & 1) + d;
        v[d] = kx < a.kw ? (int)(wr[kx] & cmask) : 0;
      }
    }
  } else {
    constexpr int BLK = Blk<B>::bytes;
    if (kb < geo.kb_total) {
      const uint8_t *p = kb < geo.kb_main
                             ? a.w + ((int64_t)g * a.cout + k) * geo.w_ch + (int64_t)kb * BLK
                             : a.proj_w + ((int64_t)gd * a.cout + k) * geo.pw_ch +
                                   (int64_t)(kb - geo.kb_main) * BLK;
      v = load_weight_unit<B>(p, u);
      if constexpr (B == 8) {
        if (a.w_bits == 6)  // 6-bit codes stored one per byte: sign-extend from bit 5
#pragma unroll
          for (int d = 0; d < 4; ++d) v[d] = (int)sext_bytes<6>((uint32_t)v[d]);
      }
    }
  }
  return v;
}

// Weights -> [G][cout/32][kb_total][j][half][ch][16 B] int8, one thread per
// 16-byte operand chunk.  The projection K-blocks of source group g hold the
// projection filter of its destination group (g + s) mod G.
template <int B, bool STEM>
__global__ void prepack_kernel(ConvArgs a, Geo geo, uint8_t *wp) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int nc32 = a.cout / 32;
  const int64_t total = (int64_t)a.in.groups * nc32 * geo.kb_total * 128;
  if (t >= total) return;
  const int within = (int)(t & 127);
  const int64_t rest = t >> 7;
  const int kb = (int)(rest % geo.kb_total);
  const int64_t r2 = rest / geo.kb_total;
  const int cblk = (int)(r2 % nc32);
  const int g = (int)(r2 / nc32);
  const int j = within >> 6, half = (within >> 5) & 1, ch = within & 31;
  const int gd = (g + a.shuffle) % a.in.groups;
  *(v4i *)(wp + t * 16) = weight_unit<B, STEM>(a, geo, g, gd, cblk * 32 + ch, kb, 2 * half + j);
}

// Geo::acc0 of an unsigned 6/8-bit layer: 128 times the sum of each output
// channel's weights (sign-extended from w_bits), one thread per channel.
__global__ void wsum_kernel(ConvArgs a, Geo geo, int32_t *acc0) {
  const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= (int64_t)a.in.groups * a.cout) return;
  const int sh = 8 - a.w_bits;
  auto wsum = [&](const int8_t *w, int K) {
    int32_t sum = 0;
    for (int k = 0; k < K; ++k) sum += (int32_t)(int8_t)(w[k] << sh) >> sh;
    return sum;
  };
  int32_t sum = wsum((const int8_t *)(a.w + c * geo.w_ch), a.kh * a.kw * a.in.cpg);
  if (a.proj.data) {  // the fused projection of destination group (g + s) mod G (its inputs get the same flip)
    const int g = (int)(c / a.cout), k = (int)(c % a.cout), gd = (g + a.shuffle) % a.in.groups;
    sum += wsum((const int8_t *)(a.proj_w + ((int64_t)gd * a.cout + k) * geo.pw_ch), a.proj.cpg);
  }
  acc0[c] = 128 * sum;
}

// FP4 (E2M1) weight slabs for the 2-bit grouped tile kernel, one MFMA
// (32 x 32 x 64) per K-block: [G][cout/32][kb_total][half][ch][16 B].
// Nibble n (word q = n / 8, position j = n % 8) of lane (ch, half) holds the
// K-block's weight code 32 half + 16 (q >> 1) + 2 j + (q & 1) as E2M1 of w / 2
// (-1, -0.5, 0, 0.5 for w = -2, -1, 0, 1); the activation unpack puts the
// same code index there (as c / 2), so every product is exact and carries a
// factor 1/4.  One thread per 16-byte lane operand.
constexpr int kSlab4 = 1024;
constexpr int kSlab6 = 1536;
__global__ void prepack_fp4_kernel(ConvArgs a, Geo geo, uint8_t *wp) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int nc32 = a.cout / 32;
  const int64_t total = (int64_t)a.in.groups * nc32 * geo.kb_total * 64;
  if (t >= total) return;
  const int within = (int)(t & 63);
  const int64_t rest = t >> 6;
  const int kb = (int)(rest % geo.kb_total);
  const int64_t r2 = rest / geo.kb_total;
  const int cblk = (int)(r2 % nc32);
  const int g = (int)(r2 / nc32);
  const int half = within >> 5, k = cblk * 32 + (within & 31);
  const int gd = (g + a.shuffle) % a.in.groups;
  const uint8_t *p = kb < geo.kb_main ? a.w + ((int64_t)g * a.cout + k) * geo.w_ch + (int64_t)kb * 16
                                      : a.proj_w + ((int64_t)gd * a.cout + k) * geo.pw_ch + (int64_t)(kb - geo.kb_main) * 16;
  const uint32_t u[2] = {((const uint32_t *)p)[2 * half], ((const uint32_t *)p)[2 * half + 1]};
  uint32_t o[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint32_t src = u[q >> 1] >> (2 * (q & 1));
    uint32_t w = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint32_t c = (src >> (4 * j)) & 3u;               // 2-bit two's complement code
      w |= ((0x9A10u >> (4 * c)) & 15u) << (4 * j);           // 0 -> 0, 1 -> 0.5, -2 -> -1, -1 -> -0.5
    }
    o[q] = w;
  }
  *(uint4 *)(wp + t * 16) = make_uint4(o[0], o[1], o[2], o[3]);
}

// FP6 (E2M3) weight slabs for 3-bit grouped layers, one MFMA (32 x 32 x 64)
// per K-block: [G][cout/32][kb_total][1536 B], a slab holding bytes 0-15 of
// every lane's 24-byte operand (lane l at 16 l), then bytes 16-23 (at
// 1024 + 8 l).  Field f (bits 6f .. 6f + 5 of the 192-bit operand) of lane
// (ch, half) holds E2M3 of the weight w of code 32 half + fp6_code(f) of the
// K-block, exact for w in -4 .. 3; the activation operand (fp6_operand)
// puts the same code there as the subnormal c / 8, so every product is exact
// and carries a factor 1/8.
// K order inside a 32-code chunk: the fields of output word 3 u + d (u: the
// chunk's low word) take the codes 16 u + 3 m + r(d) (r = 0, 2, 1 for d = 0,
// 1, 2), whose low bits the word can mask out of the low word in place.
__host__ __device__ inline int fp6_code(int f) {
  constexpr int kPerm[16] = {0, 3, 6, 9, 12, 15, 2, 5, 8, 11, 14, 1, 4, 7, 10, 13};
  return (f & 16) + kPerm[f & 15];
}
__global__ void prepack_fp6_kernel(ConvArgs a, Geo geo, uint8_t *wp) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int nc32 = a.cout / 32;
  const int64_t total = (int64_t)a.in.groups * nc32 * geo.kb_total * 64;
  if (t >= total) return;
  const int lane = (int)(t & 63);
  const int64_t rest = t >> 6;
  const int kb = (int)(rest % geo.kb_total);
  const int64_t r2 = rest / geo.kb_total;
  const int cblk = (int)(r2 % nc32);
  const int g = (int)(r2 / nc32);
  const int half = lane >> 5, k = cblk * 32 + (lane & 31);
  // the K-block's chunk of this lane half: low words, then the bit-2 word
  const uint32_t *c = (const uint32_t *)(a.w + ((int64_t)g * a.cout + k) * geo.w_ch + (int64_t)kb * 24 + 12 * half);
  const uint32_t lo0 = c[0], lo1 = c[1], hi = c[2];
  uint32_t o[6] = {0, 0, 0, 0, 0, 0};
  for (int f = 0; f < 32; ++f) {
    const int j = fp6_code(f);
    const uint32_t v = (((j < 16 ? lo0 : lo1) >> (2 * (j & 15))) & 3u) | (((hi >> b3_hi_pos(j)) & 1u) << 2);
    // E2M3 (sign, 2 exponent bits with bias 1, 3 mantissa bits) of the
    // two's complement code v: 0, 1, 2, 3, -4, -3, -2, -1
    constexpr uint32_t kE2M3[8] = {0x00, 0x08, 0x10, 0x14, 0x38, 0x34, 0x30, 0x28};
    const uint32_t e = kE2M3[v];
    const int bit = 6 * f;
    o[bit >> 5] |= e << (bit & 31);
    if ((bit & 31) > 26) o[(bit >> 5) + 1] |= e >> (32 - (bit & 31));
  }
  uint8_t *slab = wp + (t >> 6) * kSlab6;
  *(uint4 *)(slab + lane * 16) = make_uint4(o[0], o[1], o[2], o[3]);
  *(uint2 *)(slab + 1024 + lane * 8) = make_uint2(o[4], o[5]);
}

// MFMA operand of a lane's 32-code chunk (x: low words 0, 1 and the bit-2
// word) as E2M3 subnormals c / 8, fields in the fp6_code order: word 3 u + d
// = low word u masked to its fields' code pairs, or'ed with the bit-2 word
// rotated so that bit 2 of each of those codes lands two bits above its pair
// (codes 0-15 sit at even bits: rotate by 2; codes 16-31 at odd bits: by 1).
__device__ inline v8i fp6_operand(uint32_t lo0, uint32_t lo1, uint32_t hi) {
  const uint32_t r0 = __builtin_amdgcn_alignbit(hi, hi, 30), r1 = __builtin_amdgcn_alignbit(hi, hi, 31);
  v8i d;
  d[0] = (int)((lo0 & 0xC30C30C3u) | (r0 & 0x04104104u));
  d[1] = (int)((lo0 & 0x30C30C30u) | (r0 & 0x41041041u));
  d[2] = (int)((lo0 & 0x0C30C30Cu) | (r0 & 0x10410410u));
  d[3] = (int)((lo1 & 0xC30C30C3u) | (r1 & 0x04104104u));
  d[4] = (int)((lo1 & 0x30C30C30u) | (r1 & 0x41041041u));
  d[5] = (int)((lo1 & 0x0C30C30Cu) | (r1 & 0x10410410u));
  d[6] = 0;
  d[7] = 0;
  return d;
}

// Buffer resource over `bytes` bytes at `base`: loads at an offset >= bytes
// return zero (hardware range check), which implements the zero padding of
// out-of-image taps and of pixels past the end without branches.
__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void *base, int64_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc((void *)base, (short)0, (int)bytes, 0x00020000);
}
constexpr uint32_t kOob = 0x40000000u;  // offset past any tensor these kernels accept (< 2^30 B)

template <int B>
__device__ inline RawT<B, false> buf_half(__amdgpu_buffer_rsrc_t r, uint32_t voff, int soff) {
  RawT<B, false> x;
  if constexpr (B == 2) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, (int)voff, soff, 0);
    const uint2 u = __builtin_bit_cast(uint2, v);
    x.w[0] = u.x; x.w[1] = u.y;
  } else if constexpr (B == 4) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, soff, 0);
    const uint4 u = __builtin_bit_cast(uint4, v);
    x.w[0] = u.x; x.w[1] = u.y; x.w[2] = u.z; x.w[3] = u.w;
  } else if constexpr (B == 8) {
    const uint4 u0 = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, soff, 0));
    const uint4 u1 = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, soff + 16, 0));
    x.w[0] = u0.x; x.w[1] = u0.y; x.w[2] = u0.z; x.w[3] = u0.w;
    x.w[4] = u1.x; x.w[5] = u1.y; x.w[6] = u1.z; x.w[7] = u1.w;
  } else {
    const auto v = __builtin_amdgcn_raw_buffer_load_b96(r, (int)voff, soff, 0);
    x.w[0] = v[0]; x.w[1] = v[1]; x.w[2] = v[2];
  }
  return x;
}

// floor(m / d) for 0 <= m < 2^24, d >= 1, from a float estimate corrected
// by one step each way (the estimate is off by at most one).
__device__ inline int fdiv(int m, int d, float inv_d) {
  int q = (int)((float)m * inv_d);
  const int r = m - q * d;
  q -= r < 0 ? 1 : 0;
  q += r >= d ? 1 : 0;
  return q;
}

// Workgroup prologue shared by both kernels: copy the channel block's
// prepacked weights (all K-blocks) and its requant constants into LDS.
template <int CB>
__device__ inline void stage_block(const ConvArgs &a, const Geo &geo, int g, uint8_t *lds) {
  const int KB = geo.kb_total;
  const uint8_t *wsrc = geo.wp + (int64_t)(g * (a.cout / 32) + blockIdx.y * CB) * KB * kSlab;
  const int chunks = KB * CB * 128;
  for (int c = threadIdx.x; c < chunks; c += kNW * 64) {
    const int kb = c / (CB * 128);
    const int cb = (c >> 7) % CB;
    *(uint4 *)(lds + c * 16) = *(const uint4 *)(wsrc + ((int64_t)cb * KB + kb) * kSlab + (c & 127) * 16);
  }
  RqConst *rq = (RqConst *)(lds + KB * CB * kSlab);
  const int c0 = g * a.cout + blockIdx.y * CB * 32;
  for (int c = threadIdx.x; c < CB * 32; c += kNW * 64) rq[c] = geo.rq[c0 + c];
  __syncthreads();
}

// ---------------------------------------------------------------- epilogue
// Requant (+ shortcut) of one wave's CB x PB accumulator blocks and the
// store through the cyclic permutation.  Block (cb, pb) covers channels
// ch0 + 32 cb .. + 31 (rows of the MFMA output: lane holds rows
// 8 (r / 4) + 4 half + r % 4) of pixels mbase + 32 pb + lane % 32.
// RB: 2 = 2-bit identity shortcut prefetched into rw; -1 = identity shortcut
// of other widths read here; 0 = none.
template <int CB, int PB, int RB>
__device__ __forceinline__ void epilogue(const ConvArgs &a, const Geo &geo, v16i (&acc)[CB][PB], const uint32_t (&rw)[CB][PB][2],
                                int64_t mbase, int g, int gd, int ch0, int l32, int half, const RqConst *rq) {
  const int bo = store_bits(a.out.bits);  // 6-bit codes are stored as bytes
  const int qmax = (1 << a.out.bits) - 1;
  const int64_t outC = (int64_t)a.in.groups * a.cout;
  const int lsc = geo.scale == 16 ? 4 : 0;
  const bool exact64 = ((const int32_t *)(geo.rq + (int64_t)a.in.groups * a.cout))[0] != 0;
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    const int kc = ch0 + cb * 32;
    const int csb = g * a.cout + kc;
    const int cdb = gd * a.cout + kc;
    uint32_t qv[PB][4], hq[PB][4];
#pragma unroll
    for (int qi = 0; qi < 4; ++qi) {
      // keep the scheduler from hoisting every quad's constants to the top
      // (that would hold 8 quads x 16 VGPRs of fp64 constants at once)
      __builtin_amdgcn_sched_barrier(0);
      const int cq = 8 * qi + 4 * half;
      v4i rmu = {0, 0, 0, 0};
      if constexpr (RB != 0) rmu = *(const v4i *)(a.res_mult + csb + cq);
      RqConst k[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) k[e] = rq[cb * 32 + cq + e];
#pragma unroll
      for (int pb = 0; pb < PB; ++pb) {
        const int64_t mp = mbase + pb * 32 + l32;
        int32_t v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = acc[cb][pb][4 * qi + e];
        if constexpr (RB == 2) {
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] += (rmu[e] * chunk_code(rw[cb][pb], cq + e, 2)) << lsc;
        } else if constexpr (RB < 0) {
          int rc[4];
          row_quad(a.res.data + (mp < geo.M ? mp : 0) * a.res.pixel + (int64_t)gd * a.res.gstride, kc + cq,
                   a.res.bits, rc);
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] += (rmu[e] * rc[e]) << lsc;
        }
        uint32_t qword = 0, hword = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          int q;
          if (!exact64) {
            q = (int)__builtin_fma((double)v[e], k[e].s, k[e].o);
            q = min(max(q, 0), qmax);
          } else {
            const int cs = csb + cq + e;
            q = requant_mul((int64_t)(v[e] >> lsc) + (a.bias ? a.bias[cs] : 0), a.mult[cs], a.shift[cs], qmax);
          }
          if (bo == 3) {
            qword |= (uint32_t)(q & 3) << (2 * e);
            hword |= (uint32_t)((q >> 2) & 1) << (2 * e);
          } else {
            qword |= (uint32_t)q << (bo * e);
          }
        }
        qv[pb][qi] = qword;
        hq[pb][qi] = hword;
        if (a.acc_dump && mp < geo.M) {
          const v4i dv = {acc[cb][pb][4 * qi] >> lsc, acc[cb][pb][4 * qi + 1] >> lsc,
                          acc[cb][pb][4 * qi + 2] >> lsc, acc[cb][pb][4 * qi + 3] >> lsc};
          *(v4i *)(a.acc_dump + mp * outC + cdb + cq) = dv;
        }
      }
    }
    // exchange quads with the partner lane (half ^ 1) and store
#pragma unroll
    for (int pb = 0; pb < PB; ++pb) {
      const int64_t mp = mbase + pb * 32 + l32;
      const uint32_t s0 = half ? qv[pb][0] : qv[pb][2];
      const uint32_t s1 = half ? qv[pb][1] : qv[pb][3];
      const uint32_t r0 = (uint32_t)__shfl_xor((int)s0, 32);
      const uint32_t r1 = (uint32_t)__shfl_xor((int)s1, 32);
      uint32_t Q[4];
      if (half == 0) { Q[0] = qv[pb][0]; Q[1] = r0; Q[2] = qv[pb][1]; Q[3] = r1; }
      else           { Q[0] = r0; Q[1] = qv[pb][2]; Q[2] = r1; Q[3] = qv[pb][3]; }
      uint32_t hpart = 0;
      if (bo == 3) {
#pragma unroll
        for (int qi = 0; qi < 4; ++qi)  // channel 8 qi + 4 half + e at bit 2 (c & 15) + (c >> 4)
          hpart |= hq[pb][qi] << (16 * (qi & 1) + 8 * half + (qi >> 1));
        hpart |= (uint32_t)__shfl_xor((int)hpart, 32);
      }
      if (mp >= geo.M) continue;
      uint8_t *orow = a.out.data + mp * a.out.pixel + (int64_t)gd * a.out.gstride;
      if (bo == 3) {
        uint32_t *cw = (uint32_t *)orow + (int64_t)(kc >> 5) * 3;
        cw[half] = Q[0] | (Q[1] << 8) | (Q[2] << 16) | (Q[3] << 24);
        if (half == 0) cw[2] = hpart;
      } else {
        uint32_t *cw = (uint32_t *)orow + (int64_t)(kc >> 5) * bo + half * (bo / 2);
        if (bo == 2) {
          cw[0] = Q[0] | (Q[1] << 8) | (Q[2] << 16) | (Q[3] << 24);
        } else if (bo == 4) {
          *(uint2 *)cw = make_uint2(Q[0] | (Q[1] << 16), Q[2] | (Q[3] << 16));
        } else {
          *(uint4 *)cw = make_uint4(Q[0], Q[1], Q[2], Q[3]);
        }
      }
    }
  }
}

typedef double dbl2 __attribute__((ext_vector_type(2)));

// Output width BO is a compile-time constant here; fma -> saturating
// unsigned conversion (negative values and NaN give 0, which is the ReLU
// clamp) -> min with 2^BO - 1 -> shift into the quad's word.  BO = 3: the
// quad's low bit pairs form the 2-bit word as for BO = 2 and its bit 2 go
// to the chunk's bit-2 word (the two lane halves' parts or'ed together).
// AccV = v16f: the FP4 tile kernel's accumulator, t / 4 held exactly (the
// constants carry the factor 4); its shortcut term rm c / 4 is added in
// fp32, exact because the layer's |t| + 3 |rm| stays below 2^24 (a multiple
// of 1/4 below 2^22 fits the 24-bit significand).
// LAZY (2-bit shortcut, PB = 2): rw is unused; each channel block's shortcut
// words are read from LDS at rwl + 8 cb (pixel block 0) and + rws (pixel
// block 1) when that block is processed, which keeps fewer registers live.
// F32 (FP4 accumulator, 2-bit outputs): the accumulator already holds
// (t + bias) / 4 and scf[c] is the channel's fp32 scale M 2^(2 - sh); the
// requant is min(trunc(fma(v, scf, 1/2)), 3), exact under the bounds
// requant_prep_f32_kernel checks (rq is then unused); rm holds the shortcut
// scales res_mult / 4 as fp32 bits.
template <int BO, int CB, int PB, int RB, typename AccV, bool LAZY = false, bool F32 = false>
__device__ __forceinline__ void epilogue_fast_bo(const ConvArgs &a, const Geo &geo, AccV (&acc)[CB][PB],
                                        const uint32_t (&rw)[CB][PB][2], int64_t mbase, int g, int gd, int ch0,
                                        int l32, int half, const RqConst *rq, const int32_t *rm,
                                        uint32_t rwl = 0, uint32_t rws = 0, const float *scf = nullptr) {
  static_assert(!LAZY || PB == 2 || PB == 4, "lazy shortcut reads are written for two or four pixel blocks");
  static_assert(!F32 || (BO == 2 && std::is_same<AccV, v16f>::value), "the fp32 requant takes FP4 accumulators");
  constexpr int bo = BO;
  // BO = 8 also stores 6-bit codes (one per byte), clamped at 63
  const uint32_t qmax = BO == 8 ? (1u << a.out.bits) - 1u : (1u << BO) - 1u;
  const int lsc = geo.scale == 16 ? 4 : 0;
  // requant constants (and shortcut multipliers) of quad j = 4 cb + qi,
  // read one quad ahead of their use so that their LDS latency overlaps
  // the previous quad's arithmetic
  auto quad_consts = [&](int j, dbl2 (&k)[4], v4f &kf, v4i &rmu) __attribute__((always_inline)) {
    const int c0 = (j >> 2) * 32 + 8 * (j & 3) + 4 * half;
    if constexpr (F32) {
      kf = *(const v4f *)(scf + c0);
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) k[e] = dbl2{rq[c0 + e].s, rq[c0 + e].o};
    }
    rmu = v4i{0, 0, 0, 0};
    if constexpr (RB != 0) rmu = *(const v4i *)(rm + c0);
  };
  dbl2 k_cur[4];
  v4f kf_cur;
  v4i rmu_cur;
  quad_consts(0, k_cur, kf_cur, rmu_cur);
  // 2-bit codes of two channel blocks and an even number of pixel blocks:
  // each lane gathers its pixel's 64 channels (16 bytes) and stores them at
  // once; w2[cb][pb] holds the lane's 16 channels of block (cb, pb)
  constexpr bool ST16 = BO == 2 && CB == 2 && PB % 2 == 0;
  uint32_t w2[CB][PB];
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    const int kc = ch0 + cb * 32;
    uint32_t qv[PB][4];
    uint32_t hv[PB][4];
    uint32_t rwc[PB][2];
    if constexpr (RB == 2 && LAZY && PB == 2) {
      uint2 r0, r1;
      asm volatile(
          "ds_read_b64 %0, %2\n\t"
          "ds_read_b64 %1, %3\n\t"
          "s_waitcnt lgkmcnt(0)"
          : "=&v"(r0), "=&v"(r1)
          : "v"(rwl + 8 * cb), "v"(rwl + 8 * cb + rws));
      rwc[0][0] = r0.x; rwc[0][1] = r0.y;
      rwc[1][0] = r1.x; rwc[1][1] = r1.y;
    } else if constexpr (RB == 2 && LAZY) {
      uint2 r[4];
      asm volatile(
          "ds_read_b64 %0, %4\n\t"
          "ds_read_b64 %1, %5\n\t"
          "ds_read_b64 %2, %6\n\t"
          "ds_read_b64 %3, %7\n\t"
          "s_waitcnt lgkmcnt(0)"
          : "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2]), "=&v"(r[3])
          : "v"(rwl + 8 * cb), "v"(rwl + 8 * cb + rws), "v"(rwl + 8 * cb + 2 * rws), "v"(rwl + 8 * cb + 3 * rws));
#pragma unroll
      for (int pb = 0; pb < PB; ++pb) { rwc[pb][0] = r[pb & 3].x; rwc[pb][1] = r[pb & 3].y; }
    } else {
#pragma unroll
      for (int pb = 0; pb < PB; ++pb) { rwc[pb][0] = rw[cb][pb][0]; rwc[pb][1] = rw[cb][pb][1]; }
    }
#pragma unroll
    for (int qi = 0; qi < 4; ++qi) {
      // one quad at a time: without this the scheduler hoists the constant
      // loads of every quad above the last MFMAs and runs out of registers
      __builtin_amdgcn_sched_barrier(0);
      const int cq = 8 * qi + 4 * half;
      dbl2 k[4];
      v4f kf = kf_cur;
      v4i rmu;
#pragma unroll
      for (int e = 0; e < 4; ++e) k[e] = k_cur[e];
      rmu = rmu_cur;
      if (4 * cb + qi + 1 < 4 * CB) quad_consts(4 * cb + qi + 1, k_cur, kf_cur, rmu_cur);
#pragma unroll
      for (int pb = 0; pb < PB; ++pb) {
        constexpr bool FACC = std::is_same<AccV, v16f>::value;
        typename std::conditional<FACC, float, int32_t>::type v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = acc[cb][pb][4 * qi + e];
        if constexpr (RB == 2 && FACC) {
          // F32: rm holds res_mult / 4 as fp32 bits (each element copied to
          // a scalar first: a bit cast of a vector element would read the
          // vector's first element)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int32_t ri = rmu[e];
            v[e] = __builtin_fmaf(F32 ? __builtin_bit_cast(float, ri) : (float)ri * 0.25f,
                                  (float)chunk_code(rwc[pb], cq + e, 2), v[e]);
          }
        } else if constexpr (RB == 2) {
          // |res_mult| < 2^15 and codes < 4: 24-bit signed products
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] += __mul24(rmu[e] << lsc, chunk_code(rwc[pb], cq + e, 2));
        } else if constexpr (RB < 0) {
          const int64_t mp = mbase + pb * 32 + l32;
          int rc[4];
          row_quad(a.res.data + (mp < geo.M ? mp : 0) * a.res.pixel + (int64_t)gd * a.res.gstride, kc + cq,
                   a.res.bits, rc);
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] += (rmu[e] * rc[e]) << lsc;
        }
        uint32_t qword = 0, hword = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          uint32_t q;
          if constexpr (F32) {
            const float y = __builtin_fmaf((float)v[e], kf[e], 0.5f);
            asm("v_cvt_u32_f32 %0, %1" : "=v"(q) : "v"(y));
          } else {
            const double d = __builtin_fma((double)v[e], k[e].x, k[e].y);
            asm("v_cvt_u32_f64 %0, %1" : "=v"(q) : "v"(d));
          }
          if constexpr (BO == 3) {
            const uint32_t qq = min(q, qmax);
            qword |= (qq & 3u) << (2 * e);
            hword |= (qq >> 2) << (2 * e);
          } else {
            qword |= min(q, qmax) << (bo * e);
          }
        }
        qv[pb][qi] = qword;
        hv[pb][qi] = hword;
      }
    }
#pragma unroll
    for (int pb = 0; pb < PB; ++pb) {
      const int64_t mp = mbase + pb * 32 + l32;
      // v_permlane32_swap exchanges the upper lane half of its first
      // operand with the lower lane half of its second; afterwards every
      // lane holds words 0, 1 (and 2, 3) of its 32 channels in order
      const auto p0 = __builtin_amdgcn_permlane32_swap(qv[pb][0], qv[pb][2], false, false);
      const auto p1 = __builtin_amdgcn_permlane32_swap(qv[pb][1], qv[pb][3], false, false);
      const uint32_t Q[4] = {p0[0], p0[1], p1[0], p1[1]};
      if constexpr (BO == 3) {
        // bit 2 of channel c = 8 qi + 4 half + e at bit 2 (c & 15) + (c >> 4)
        uint32_t hp = 0;
#pragma unroll
        for (int qi = 0; qi < 4; ++qi) hp |= hv[pb][qi] << (16 * (qi & 1) + 8 * half + (qi >> 1));
        const auto hs = __builtin_amdgcn_permlane32_swap(hp, hp, false, false);
        const uint32_t hw = hs[0] | hs[1];
        if (mp >= geo.M) continue;
        uint32_t *cw = (uint32_t *)(a.out.data + mp * a.out.pixel + (int64_t)gd * a.out.gstride) + (int64_t)(kc >> 5) * 3;
        cw[half] = Q[0] | (Q[1] << 8) | (Q[2] << 16) | (Q[3] << 24);
        if (half == 0) cw[2] = hw;
        continue;
      }
      if constexpr (ST16) {
        w2[cb][pb] = Q[0] | (Q[1] << 8) | (Q[2] << 16) | (Q[3] << 24);
        continue;
      }
      if (mp >= geo.M) continue;
      uint32_t *cw = (uint32_t *)(a.out.data + mp * a.out.pixel + (int64_t)gd * a.out.gstride) +
                     (int64_t)(kc >> 5) * bo + half * (bo / 2);
      if (bo == 2) {
        cw[0] = Q[0] | (Q[1] << 8) | (Q[2] << 16) | (Q[3] << 24);
      } else if (bo == 4) {
        *(uint2 *)cw = make_uint2(Q[0] | (Q[1] << 16), Q[2] | (Q[3] << 16));
      } else {
        *(uint4 *)cw = make_uint4(Q[0], Q[1], Q[2], Q[3]);
      }
    }
  }
  if constexpr (ST16) {
    // pixel blocks 2 i and 2 i + 1: lanes of half 0 take block 2 i, lanes of
    // half 1 block 2 i + 1; per channel block the swap brings the other
    // half's 16 channels of that pixel (words ordered cb, half as stored)
#pragma unroll
    for (int i = 0; i < PB / 2; ++i) {
      const auto s0 = __builtin_amdgcn_permlane32_swap(w2[0][2 * i], w2[0][2 * i + 1], false, false);
      const auto s1 = __builtin_amdgcn_permlane32_swap(w2[1][2 * i], w2[1][2 * i + 1], false, false);
      const int64_t mp = mbase + (2 * i + half) * 32 + l32;
      if (mp >= geo.M) continue;
      uint8_t *dst = a.out.data + mp * a.out.pixel + (int64_t)gd * a.out.gstride + (int64_t)(ch0 >> 5) * 8;
      *(uint4 *)dst = make_uint4(s0[0], s0[1], s1[0], s1[1]);
    }
  }
}

// rq: requant constants from the wave's first channel on; rm: the shortcut
// multipliers of the same channels (used with a shortcut only).
template <int CB, int PB, int RB>
__device__ __forceinline__ void epilogue_fast(const ConvArgs &a, const Geo &geo, v16i (&acc)[CB][PB],
                                     const uint32_t (&rw)[CB][PB][2], int64_t mbase, int g, int gd, int ch0,
                                     int l32, int half, const RqConst *rq, const int32_t *rm) {
  if (a.out.bits == 2)
    epilogue_fast_bo<2, CB, PB, RB>(a, geo, acc, rw, mbase, g, gd, ch0, l32, half, rq, rm);
  else if (a.out.bits == 4)
    epilogue_fast_bo<4, CB, PB, RB>(a, geo, acc, rw, mbase, g, gd, ch0, l32, half, rq, rm);
  else  // 6 or 8
    epilogue_fast_bo<8, CB, PB, RB>(a, geo, acc, rw, mbase, g, gd, ch0, l32, half, rq, rm);
}

// Each kernel is built twice: GEN = false carries only the fast epilogue
// (and so needs far fewer registers), GEN = true the general one.
template <int CB, int PB, int RB, bool GEN>
__device__ inline void finish_tile(const ConvArgs &a, const Geo &geo, v16i (&acc)[CB][PB],
                                   const uint32_t (&rw)[CB][PB][2], int64_t mbase, int g, int gd, int ch0,
                                   int l32, int half, const uint8_t *lds) {
  const RqConst *rq = (const RqConst *)(lds + geo.kb_total * CB * kSlab);
  if constexpr (GEN) epilogue<CB, PB, RB>(a, geo, acc, rw, mbase, g, gd, ch0, l32, half, rq);
  else epilogue_fast<CB, PB, RB>(a, geo, acc, rw, mbase, g, gd, ch0, l32, half, rq,
                                 a.res_mult + (int64_t)g * a.cout + ch0);
}

// The layer's int64-requant flag (written by requant_prep_kernel after its
// constants): set when some channel's fp64 requant could be inexact.
__device__ inline bool int64_flag(const ConvArgs &a, const Geo &geo) {
  return ((const int32_t *)(geo.rq + (int64_t)a.in.groups * a.cout))[0] != 0;
}

// Whether a layer needs the general epilogue: the int64 requant fallback,
// the accumulator dump, 3-bit outputs or an identity shortcut of other than
// 2 bits.  Uniform.
__device__ inline bool needs_general(const ConvArgs &a, const Geo &geo, int rb) {
  return int64_flag(a, geo) || a.acc_dump != nullptr || a.out.bits == 3 || rb < 0;
}

// Whether this build of a persistent kernel leaves at once.  a.gated: the
// launch is the general partner of a tiled launch (which covers every case
// but the int64 requant), so only the general build runs, and only when the
// flag is set; otherwise the fast and the general build split by
// needs_general.
__device__ inline bool skip_build(const ConvArgs &a, const Geo &geo, int rb, bool gen) {
  if (a.gated) return !gen || !int64_flag(a, geo);
  return needs_general(a, geo, rb) != gen;
}

// Loads of the K loop, the LDS operand reads and the MFMAs of one K-block
// are the same for both kernels; the loader differs.  Three activation
// slots rotate: K-block kb uses one slot and refills another with K-block
// kb + 2, which may already belong to the wave's next tile.  PALQ_KLOOP walks
// one tile starting with the slots in (A, B, C) order (A holds K-block 0, B
// K-block 1); the three call orders keep every slot in fixed registers.  The
// weight operands of a K-block are read from LDS at its start; the
// activation unpack covers most of that latency.
#define PALQ_KLOOP_BODY(KBI, XU, XF)                                                             \
  {                                                                                               \
    v4i wu[2][CB];                                                                                \
    read_w(KBI, wu);                                                                              \
    load_next(XF);                                                                                \
    _Pragma("unroll") for (int j = 0; j < 2; ++j) {                                               \
      v4i bop[PB];                                                                                \
      _Pragma("unroll") for (int pb = 0; pb < PB; ++pb) bop[pb] = operand(XU[pb], j);             \
      _Pragma("unroll") for (int cb = 0; cb < CB; ++cb)                                           \
          _Pragma("unroll") for (int pb = 0; pb < PB; ++pb) acc[cb][pb] =                         \
              __builtin_amdgcn_mfma_i32_32x32x32_i8(wu[j][cb], bop[pb], acc[cb][pb], 0, 0, 0);    \
    }                                                                                             \
  }

#define PALQ_KLOOP(XA, XB, XC)                                  \
  {                                                             \
    int kb = 0;                                                 \
    for (; kb + 3 <= KB; kb += 3) {                             \
      PALQ_KLOOP_BODY(kb, XA, XC)                               \
      PALQ_KLOOP_BODY(kb + 1, XB, XA)                           \
      PALQ_KLOOP_BODY(kb + 2, XC, XB)                           \
    }                                                           \
    if (kb < KB) PALQ_KLOOP_BODY(kb, XA, XC)                    \
    if (kb + 1 < KB) PALQ_KLOOP_BODY(kb + 1, XB, XA)            \
  }

// ---------------------------------------------------------------- grouped kernel
// Grouped B-bit conv.  Persistent workgroups of kNW waves keep the whole K
// extent of CB x 32 output channels of one group resident in LDS (one
// barrier, at the start); each wave then walks its own tiles of PB x 32 output
// pixels.  Per K-block a lane issues one buffer load per pixel block (its
// pixel's 32 codes of the current tap and 64-code block), two K-blocks ahead
// of use and across tile boundaries; the weight operands are read from LDS
// two K-blocks ahead too.
template <int B, int CB, int PB, int RB, bool GEN>
__global__ __launch_bounds__(kNW * 64) void conv_grouped_kernel(ConvArgs a, Geo geo, int tiles) {
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  constexpr int BLK = Blk<B>::bytes;
  using Raw = RawT<B, false>;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int l32 = lane & 31;
  const int half = lane >> 5;
  const int G = a.in.groups;
  const int g = blockIdx.z;
  const int gd = (g + a.shuffle) % G;
  const int ch0 = blockIdx.y * CB * 32;
  const int KB = geo.kb_total;

  // the launcher may start both builds when it cannot tell which applies:
  // the other one leaves at once (before any barrier)
  if (skip_build(a, geo, RB, GEN)) return;
  stage_block<CB>(a, geo, g, lds);
  const int first = blockIdx.x * kNW + wave;
  const int tstride = gridDim.x * kNW;
  if (first >= tiles) return;  // no barrier follows

  const auto rin = make_rsrc(a.in.data, a.in.bytes);
  // without a projection this resource has no bytes: every load returns 0
  const auto rpj = a.proj.data ? make_rsrc(a.proj.data, a.proj.bytes)
                               : make_rsrc(a.in.data, 0);
  const int pixb = (int)a.in.pixel;
  const int rowb = a.in.w * pixb;
  const int HW = a.ho * a.wo;
  const float inv_hw = geo.inv_hw, inv_wo = geo.inv_wo;

  // ---- loader: tile lt, K-block cursor; geometry of tile lt per pixel block
  int lt = first, l_kb = 0, l_tap = 0, l_cblk = 0, l_ky = 0, l_kx = 0, l_tapoff = 0;
  int off0[PB];
  uint32_t tmask[PB], poff[PB];
  auto geometry = [&](int t) {
#pragma unroll
    for (int pb = 0; pb < PB; ++pb) {
      const int m = t * PB * 32 + pb * 32 + l32;
      const bool valid = t < tiles && m < geo.M;
      const int mm = valid ? m : 0;
      const int n = fdiv(mm, HW, inv_hw);
      const int rem = mm - n * HW;
      const int oy = fdiv(rem, a.wo, inv_wo);
      const int ox = rem - oy * a.wo;
      const int iy0 = oy * a.stride - a.pad, ix0 = ox * a.stride - a.pad;
      off0[pb] = ((n * a.in.h + iy0) * a.in.w + ix0) * pixb + g * (int)a.in.gstride + half * (BLK / 2);
      const int xlo = max(0, -ix0), xhi = min(a.kw, a.in.w - ix0);
      const uint32_t below = xhi >= 32 ? 0xffffffffu : ((1u << max(xhi, 0)) - 1u);
      const uint32_t cols = xhi > xlo ? (below & ~((1u << xlo) - 1u)) : 0u;
      const int ylo = max(0, -iy0), yhi = min(a.kh, a.in.h - iy0);
      uint32_t mk = 0;
      for (int ky = ylo; ky < yhi; ++ky) mk |= cols << (ky * a.kw);
      tmask[pb] = valid ? mk : 0u;
      poff[pb] = (a.proj.data && valid)
                     ? (uint32_t)(((n * a.proj.h + oy * a.proj_stride) * a.proj.w + ox * a.proj_stride) *
                                      (int)a.proj.pixel +
                                  gd * (int)a.proj.gstride + half * (BLK / 2))
                     : kOob;
    }
  };
  geometry(lt);
  // Every call issues exactly PB loads (K-blocks with no data read the
  // zero-returning offset), so the wait counts are static.
  auto load_next = [&](Raw (&x)[PB]) {
    if (l_kb < geo.kb_main) {
      // the per-lane offset carries the tap so that it is >= 0 whenever the
      // tap is in the image (off0 alone is negative on the top/left border);
      // only the non-negative block offset goes to soffset
      const int soff = l_cblk * BLK;
#pragma unroll
      for (int pb = 0; pb < PB; ++pb) {
        const uint32_t vo = ((tmask[pb] >> l_tap) & 1u) ? (uint32_t)(off0[pb] + l_tapoff) : kOob;
        x[pb] = buf_half<B>(rin, vo, soff);
      }
      if (++l_cblk == geo.cpb) {
        l_cblk = 0;
        ++l_tap;
        if (++l_kx == a.kw) { l_kx = 0; ++l_ky; }
        l_tapoff = l_ky * rowb + l_kx * pixb;
      }
    } else {
      const int soff = (l_kb - geo.kb_main) * BLK;
#pragma unroll
      for (int pb = 0; pb < PB; ++pb) x[pb] = buf_half<B>(rpj, poff[pb], soff);
    }
    if (++l_kb == KB) {  // move on to the wave's next tile
      l_kb = l_tap = l_cblk = l_ky = l_kx = l_tapoff = 0;
      lt += tstride;
      geometry(lt);
    }
  };
  auto read_w = [&](int kb, v4i (&aop)[2][CB]) {
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int cb = 0; cb < CB; ++cb)
        aop[j][cb] = *(const v4i *)(lds + (kb * CB + cb) * kSlab + ((j * 2 + half) * 32 + l32) * 16);
  };
  auto operand = [&](const Raw &r, int j) -> v4i { return act_operand<B>(r, j); };

  Raw xs0[PB], xs1[PB], xs2[PB];
  load_next(xs0);
  load_next(xs1);
  int phase = 0;
  const auto rres = make_rsrc(a.res.data, a.res.data ? a.res.bytes : 0);
  for (int ct = first; ct < tiles; ct += tstride) {
    // shortcut codes of this tile (2-bit): fetched now, used by the epilogue
    uint32_t rw[CB][PB][2];
#pragma unroll
    for (int cb = 0; cb < CB; ++cb)
#pragma unroll
      for (int pb = 0; pb < PB; ++pb) {
        rw[cb][pb][0] = rw[cb][pb][1] = 0;
        if constexpr (RB == 2) {
          const int m = ct * PB * 32 + pb * 32 + l32;
          const uint32_t ro = m < geo.M ? (uint32_t)(m * (int)a.res.pixel + gd * (int)a.res.gstride + ((ch0 + cb * 32) >> 5) * 8)
                                        : kOob;
          const auto v = __builtin_amdgcn_raw_buffer_load_b64(rres, (int)ro, 0, 0);
          const uint2 u = __builtin_bit_cast(uint2, v);
          rw[cb][pb][0] = u.x;
          rw[cb][pb][1] = u.y;
        }
      }
    v16i acc[CB][PB];
#pragma unroll
    for (int cb = 0; cb < CB; ++cb)
#pragma unroll
      for (int pb = 0; pb < PB; ++pb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          // row r of the 32 x 32 block is channel 8 (r / 4) + 4 half + r % 4
          if constexpr (B == 8)
            acc[cb][pb][r] = geo.acc0[(int64_t)g * a.cout + ch0 + cb * 32 + 8 * (r >> 2) + 4 * half + (r & 3)];
          else
            acc[cb][pb][r] = 0;
        }
    if (phase == 0) PALQ_KLOOP(xs0, xs1, xs2)
    else if (phase == 1) PALQ_KLOOP(xs1, xs2, xs0)
    else PALQ_KLOOP(xs2, xs0, xs1)
    phase = (phase + KB) % 3;
    finish_tile<CB, PB, RB, GEN>(a, geo, acc, rw, (int64_t)ct * PB * 32, g, gd, ch0, l32, half, lds);
  }
}

// ---------------------------------------------------------------- stem kernel
// First layer: 8-bit signed input with at most 4 channels per pixel (one
// 4-byte row), 8-bit weights, any kh and kw <= 8.  One 16-code operand unit
// is four consecutive kx taps of one filter row (pixel-major, 4 bytes each;
// the filter's padding byte is masked to 0 in the prepacked weights), a
// K-block is two filter rows.  Same persistent structure as the grouped
// kernel.
template <int CB, int PB, int RB, bool GEN>
__global__ __launch_bounds__(kNW * 64) void conv_stem_kernel(ConvArgs a, Geo geo, int tiles) {
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  using Raw = RawT<8, true>;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int l32 = lane & 31;
  const int half = lane >> 5;
  const int G = a.in.groups;
  const int g = blockIdx.z;
  const int gd = (g + a.shuffle) % G;
  const int ch0 = blockIdx.y * CB * 32;
  const int KB = geo.kb_total;

  // the launcher may start both builds when it cannot tell which applies:
  // the other one leaves at once (before any barrier)
  if (skip_build(a, geo, RB, GEN)) return;
  stage_block<CB>(a, geo, g, lds);
  const int first = blockIdx.x * kNW + wave;
  const int tstride = gridDim.x * kNW;
  if (first >= tiles) return;

  const auto rin = make_rsrc(a.in.data, a.in.bytes);
  const int pixb = (int)a.in.pixel;
  const int rowb = a.in.w * pixb;
  const int HW = a.ho * a.wo;
  const float inv_hw = geo.inv_hw, inv_wo = geo.inv_wo;

  int lt = first, l_kb = 0;
  int off0[PB], iy0[PB];
  uint32_t xmask[PB];
  auto geometry = [&](int t) {
#pragma unroll
    for (int pb = 0; pb < PB; ++pb) {
      const int m = t * PB * 32 + pb * 32 + l32;
      const bool valid = t < tiles && m < geo.M;
      const int mm = valid ? m : 0;
      const int n = fdiv(mm, HW, inv_hw);
      const int rem = mm - n * HW;
      const int oy = fdiv(rem, a.wo, inv_wo);
      const int ox = rem - oy * a.wo;
      iy0[pb] = valid ? oy * a.stride - a.pad : -(1 << 20);  // invalid pixel: every row out of range
      const int ix0 = ox * a.stride - a.pad;
      off0[pb] = ((n * a.in.h + oy * a.stride - a.pad) * a.in.w + ix0) * pixb + g * (int)a.in.gstride;
      const int xlo = max(0, -ix0), xhi = min(min(8, a.kw), a.in.w - ix0);
      const uint32_t below = (1u << max(xhi, 0)) - 1u;
      xmask[pb] = xhi > xlo ? (below & ~((1u << xlo) - 1u)) : 0u;
    }
  };
  geometry(lt);
  // Without padding (the network pads the input beforehand) every tap
  // with a non-zero weight lies inside the image: a lane's 8 taps of one
  // filter row are two 16-byte loads, with no masks (bytes past the real
  // taps, even in the next row, meet zero weights; past the tensor's end
  // they read as zero).
  const bool unpadded = a.pad == 0;
  auto load_next = [&](Raw (&x)[PB]) {
    const int ky = 2 * l_kb + half;  // this lane's filter row
    if (unpadded) {
#pragma unroll
      for (int pb = 0; pb < PB; ++pb) {
        const uint32_t vo = iy0[pb] >= 0 ? (uint32_t)(off0[pb] + ky * rowb) : kOob;
        const uint4 v0 = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rin, (int)vo, 0, 0));
        const uint4 v1 = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rin, (int)vo, 16, 0));
        x[pb].w[0] = v0.x; x[pb].w[1] = v0.y; x[pb].w[2] = v0.z; x[pb].w[3] = v0.w;
        x[pb].w[4] = v1.x; x[pb].w[5] = v1.y; x[pb].w[6] = v1.z; x[pb].w[7] = v1.w;
      }
      if (++l_kb == KB) {
        l_kb = 0;
        lt += tstride;
        geometry(lt);
      }
      return;
    }
#pragma unroll
    for (int pb = 0; pb < PB; ++pb) {
      const bool rowok = ky < a.kh && iy0[pb] + ky >= 0 && iy0[pb] + ky < a.in.h;
      const int rbase = off0[pb] + ky * rowb;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const uint32_t vo = (rowok && ((xmask[pb] >> i) & 1u)) ? (uint32_t)(rbase + i * pixb) : kOob;
        x[pb].w[i] = (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(rin, (int)vo, 0, 0);
      }
    }
    if (++l_kb == KB) {
      l_kb = 0;
      lt += tstride;
      geometry(lt);
    }
  };
  auto read_w = [&](int kb, v4i (&aop)[2][CB]) {
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int cb = 0; cb < CB; ++cb)
        aop[j][cb] = *(const v4i *)(lds + (kb * CB + cb) * kSlab + ((j * 2 + half) * 32 + l32) * 16);
  };
  auto operand = [&](const Raw &r, int j) -> v4i {
    v4i o = {(int)r.w[4 * j], (int)r.w[4 * j + 1], (int)r.w[4 * j + 2], (int)r.w[4 * j + 3]};
    return o;
  };

  Raw xs0[PB], xs1[PB], xs2[PB];
  load_next(xs0);
  load_next(xs1);
  int phase = 0;
  uint32_t rw[CB][PB][2] = {};
  for (int ct = first; ct < tiles; ct += tstride) {
    v16i acc[CB][PB];
#pragma unroll
    for (int cb = 0; cb < CB; ++cb)
#pragma unroll
      for (int pb = 0; pb < PB; ++pb)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[cb][pb][r] = 0;
    if (phase == 0) PALQ_KLOOP(xs0, xs1, xs2)
    else if (phase == 1) PALQ_KLOOP(xs1, xs2, xs0)
    else PALQ_KLOOP(xs2, xs0, xs1)
    phase = (phase + KB) % 3;
    finish_tile<CB, PB, RB, GEN>(a, geo, acc, rw, (int64_t)ct * PB * 32, g, gd, ch0, l32, half, lds);
  }
}

// ---------------------------------------------------------------- tile kernel
// Grouped 2-bit conv as a tiled implicit GEMM.  A tile is TN output channels
// x TM output pixels of one group; a workgroup's WN x WM waves each own
// CB x 32 channels x PB x 32 pixels of it.  The prepacked int8 weight slabs
// and the packed activation codes of every 64-code K-block go straight from
// memory into a ring of kStages LDS stages (buffer loads with the LDS
// destination, 16 bytes per lane, coalesced), kStages - 1 K-blocks ahead of
// the MFMAs; one barrier per K-block.  No registers hold data in flight.
// The compiler makes every ordinary read of an LDS array that such loads
// write wait for all of them, which would drain the ring at each K-block,
// so the ring's operands are read by inline asm that waits for just those
// reads; the requant constants and shortcut multipliers (of the at most two
// channel blocks a run of tiles touches) live in arrays of their own,
// staged before the first load, and a 2-bit identity shortcut's codes for a
// tile come through the load stream into one of two buffers of the ring's
// array.
//
// Workgroups are persistent: workgroup w walks a contiguous run of tiles
// (pixel tile fastest), and the fetches run across tile boundaries, so the
// next tile's first K-blocks are in flight during this tile's epilogue.
// Workgroup ids are dealt round-robin over the 8 XCDs; the runs are laid out
// so that each XCD gets one contiguous range of tiles, which keeps a group's
// weights in that XCD's L2.  Fast epilogue only: layers that need the
// general one leave at once.
#ifndef PALQ_TILE_STAGES
#define PALQ_TILE_STAGES 4
#endif
#ifndef PALQ_STEM_STAGES
#define PALQ_STEM_STAGES 3
#endif
constexpr int kStages = PALQ_TILE_STAGES;

// s_waitcnt immediates (gfx9 encoding): vmcnt(n) alone, and lgkmcnt(0) alone.
constexpr int waitcnt_vm(int n) { return (n & 15) | ((n >> 4) << 14) | 0x70 | 0xF00; }
constexpr int kWaitLgkm0 = 0xC07F;

// Barrier for the LDS ring: the caller has already waited for what must be
// complete; the empty asm statements keep the compiler from moving memory
// operations across it.
__device__ __forceinline__ void ring_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Tile order of the tiled kernel.  The npt pixel tiles are cut into nch
// chunks (1 <= nch <= npt; chunk c: tiles b_c .. b_(c+1) - 1 with
// b_c = c npt / nch); the tile index runs over chunks, then (group, channel
// block) combos, then the chunk's pixel tiles.  The workgroups of one XCD
// take a contiguous range of indices: with nch = 8 about one chunk with all
// its groups (a pixel's groups share its cache lines, which that XCD's L2
// then fetches once), with nch = 1 a few combos over all pixels (each XCD
// reads only its combos' weights).  Runs of at most npt / nch tiles touch
// at most two (chunk, combo) segments.
struct TileIt {
  int pt, combo;  // pixel tile, combo g * ncb + cbk
  int c, b, e;    // chunk and its pixel tiles b .. e - 1
};
__device__ __forceinline__ TileIt tile_at(int t, int npt, int ncombo, int nch) {
  const int u = t / ncombo;
  const int c = min(((u + 1) * nch + npt - 1) / npt - 1, nch - 1);  // last chunk with b_c <= u
  const int b = c * npt / nch, e = (c + 1) * npt / nch;
  const int r = t - ncombo * b;
  return {b + r % (e - b), r / (e - b), c, b, e};
}
// The tile after `it` in the same order (past the last: pt >= npt).
__device__ __forceinline__ void tile_next(TileIt &it, int npt, int ncombo, int nch) {
  if (++it.pt < it.e) return;
  it.pt = it.b;
  if (++it.combo < ncombo) return;
  it.combo = 0;
  ++it.c;
  it.b = it.e;
  it.pt = it.b;
  it.e = it.c < nch ? (it.c + 1) * npt / nch : npt + 1;
}

// STEM: the 8-bit first layer on an input whose zero border is explicit
// (pad 0): a K-block is two filter rows of 8 four-byte taps, 64 bytes per
// pixel, fetched as four 16-byte pieces (lane half h of the MFMA takes row
// 2 kb + h, its 8 taps being the two 16-code operand units); no unpack.
// DUMP: also write the int32 accumulators to a.acc_dump (destination channel
// order, without the operand scale).  (2-bit layers on the FP4 matrix cores
// run on conv_fp4_kernel instead.)
template <int CB, int PB, int WN, int WM, int RB, bool STEM = false, int kStages = PALQ_TILE_STAGES,
          bool DUMP = false>
__global__ __launch_bounds__(WN * WM * 64, 2) void conv_tile_kernel(ConvArgs a, Geo geo, int npt,
                                                                                      int ncb, int nch) {
  constexpr int B = 2;
  constexpr int NT = WN * WM * 64;
  constexpr int TN = WN * CB * 32, TM = WM * PB * 32;
  constexpr int BLK = STEM ? 64 : Blk<B>::bytes;  // activation bytes of one pixel's K-block
  constexpr int SLAB = kSlab;        // weight bytes of a (K-block, 32 channels)
  constexpr int WST = TN / 32 * SLAB;  // weight bytes of one K-block
  constexpr int XST = TM * BLK;       // activation bytes of one K-block
  constexpr int SSB = WST + XST;      // one K-block of a ring stage
  constexpr int SST = SSB;            // one ring stage
  constexpr int WP = WST / 16;        // 16-byte weight pieces of a K-block
  constexpr int WLD = WP / NT;       // weight loads per thread and K-block
  constexpr int XP = XST / 16;          // 16-byte activation pieces of a K-block
  constexpr bool XALL = XP >= NT;       // every thread loads (XLD pieces), else the first XP threads one
  constexpr int XLD = XALL ? XP / NT : 1;
  static_assert(WLD == 1 || WLD == 2, "weight loads per thread");
  static_assert(XP == NT / 2 || XP % NT == 0, "activation pieces");
  static_assert(!STEM || (XALL && RB == 0), "stem layout");
  static_assert(STEM || XP <= NT, "grouped layers: at most one activation piece (one pixel) per thread");
  // loads per K-block of the waves with the fewest (the ring waits on that):
  // every thread loads WLD weight pieces, the first XP threads (or all) the
  // activations
  constexpr int LPK = WLD + (XALL ? XLD : 0);
  constexpr int RQB = 2 * TN * (int)sizeof(RqConst);  // requant constants of two channel blocks
  constexpr int RMB = RB ? 2 * TN * 4 : 0;            // their shortcut multipliers
  constexpr int RPX = TN / 4;                          // shortcut code bytes per pixel of a tile
  constexpr int RSB = RB ? TM * RPX : 0;               // shortcut codes of one tile
  constexpr int RPT = RB ? RSB / (NT * 16) : 0;      // 16-byte shortcut pieces per thread
  static_assert(RB == 0 || (RPT >= 1 && RSB == RPT * NT * 16), "whole shortcut pieces per thread");
  __shared__ __attribute__((aligned(16))) uint8_t lds[kStages * SST + 2 * RSB];
  __shared__ RqConst rq_area[2 * TN];
  __shared__ int32_t rm_area[RB ? 2 * TN : 1];
  static_assert(CB == 2 && PB == 2, "compute() below is written out for 2 x 2 blocks");
  using Raw = RawT<B, false>;

  // the launcher takes 2-bit outputs and 2-bit (or no) shortcuts only; a
  // layer whose fp64 requant could be inexact runs on the general partner
  if (int64_flag(a, geo) || a.out.bits != 2 || RB < 0) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, half = lane >> 5;
  const int wn = wave / WM, wm = wave % WM;

  // This workgroup's run of tiles (tile_at: pixel tile and combo
  // g * ncb + cbk).  Workgroup id i runs on XCD x = i mod 8; XCD x takes the
  // x-th eighth of the tiles, split over its P = n / 8 workgroups in runs of
  // floor or ceil(T_x / P) (the longer runs on the lowest y = i / 8, i.e. the
  // first workgroups dispatched, one per CU), so every CU gets the same work
  // to within one tile.
  const int G = a.in.groups;
  const int T = npt * ncb * G;
  const int P = (int)gridDim.x >> 3;  // the grid is a multiple of 8
  const int x = (int)(blockIdx.x & 7), y = (int)(blockIdx.x >> 3);
  const int Tq = T >> 3, Tr = T & 7;
  const int Tx = Tq + (x < Tr ? 1 : 0);
  const int base = Tx / P, ex = Tx % P;
  const int t_begin = x * Tq + min(x, Tr) + y * base + min(y, ex);
  const int t_end = t_begin + base + (y < ex ? 1 : 0);
  if (t_begin >= t_end) return;  // no barrier yet
  const int KB = geo.kb_total;
  const int total = (t_end - t_begin) * KB;  // K-blocks this workgroup runs

  // requant constants of the run's first and last combo (slots 0 and 1; a
  // run spans at most two: the launcher keeps runs <= npt / nch tiles)
  const int combo0 = tile_at(t_begin, npt, ncb * G, nch).combo;
  const int combo1 = tile_at(t_end - 1, npt, ncb * G, nch).combo;
  for (int c = tid; c < 2 * TN; c += NT) {
    const int combo = c < TN ? combo0 : combo1;
    const int cbk = combo % ncb, g = combo / ncb;
    rq_area[c] = geo.rq[(int64_t)g * a.cout + cbk * TN + c % TN];
    if constexpr (RB != 0) rm_area[c] = a.res_mult[(int64_t)g * a.cout + cbk * TN + c % TN];
  }
  __syncthreads();
  const uint32_t lds_base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t *)lds;

  const auto rw_src = make_rsrc(geo.wp, (int64_t)G * a.cout * KB * (SLAB / 32));
  const auto rin = make_rsrc(a.in.data, a.in.bytes);
  const auto rpj = a.proj.data ? make_rsrc(a.proj.data, a.proj.bytes)
                               : make_rsrc(a.in.data, 0);
  const int pixb = (int)a.in.pixel;
  const int rowb = a.in.w * pixb;
  const int HW = a.ho * a.wo;
  const float inv_hw = geo.inv_hw, inv_wo = geo.inv_wo;

  // ---- fetcher: this thread's share of K-block f_kb of tile f_tile
  // weights: 16-byte pieces tid + i * NT of the K-block's TN/32 slabs;
  // activations: piece tid (threads < XTH), i.e. pixel xp of the tile
  const int xp = tid, xb = 0;
  typedef __attribute__((address_space(3))) void *lds_ptr;
  int f_tile = t_begin, f_kb = 0, f_tap = 0, f_cblk = 0, f_kx = 0, f_ky = 0, f_tapoff = 0;
  TileIt f_it = tile_at(t_begin, npt, ncb * G, nch);
  uint32_t wbase, tmask;
  int off0, poff;
  // stem: piece tid + i NT is quarter (tid & 3) of pixel tid / 4 + i NT / 4:
  // filter row 2 kb + ((tid >> 1) & 1), bytes 16 (tid & 1) ..
  int soff[XLD];
  auto tile_geometry = [&]() __attribute__((always_inline)) {
    const int pt = f_it.pt;
    const int cbk = f_it.combo % ncb;
    const int g = f_it.combo / ncb;
    const int gd = (g + a.shuffle) % G;
    wbase = (uint32_t)((((int64_t)g * (a.cout / 32) + cbk * (TN / 32)) * KB) * SLAB);
    if constexpr (STEM) {
#pragma unroll
      for (int i = 0; i < XLD; ++i) {
        const int m = pt * TM + (tid >> 2) + i * (NT / 4);
        const bool valid = f_tile < t_end && m < geo.M;
        const int mm = valid ? m : 0;
        const int n = fdiv(mm, HW, inv_hw);
        const int rem = mm - n * HW;
        const int oy = fdiv(rem, a.wo, inv_wo);
        const int ox = rem - oy * a.wo;
        soff[i] = valid ? ((n * a.in.h + oy * a.stride) * a.in.w + ox * a.stride) * pixb + g * (int)a.in.gstride +
                              ((tid >> 1) & 1) * rowb + (tid & 1) * 16
                        : -1;
      }
      return;
    }
    const int m = pt * TM + xp;
    const bool valid = f_tile < t_end && m < geo.M && xp < TM;
    const int mm = valid ? m : 0;
    const int n = fdiv(mm, HW, inv_hw);
    const int rem = mm - n * HW;
    const int oy = fdiv(rem, a.wo, inv_wo);
    const int ox = rem - oy * a.wo;
    const int iy0 = oy * a.stride - a.pad, ix0 = ox * a.stride - a.pad;
    off0 = ((n * a.in.h + iy0) * a.in.w + ix0) * pixb + g * (int)a.in.gstride + xb;
    const int xlo = max(0, -ix0), xhi = min(a.kw, a.in.w - ix0);
    const uint32_t below = xhi >= 32 ? 0xffffffffu : ((1u << max(xhi, 0)) - 1u);
    const uint32_t cols = xhi > xlo ? (below & ~((1u << xlo) - 1u)) : 0u;
    const int ylo = max(0, -iy0), yhi = min(a.kh, a.in.h - iy0);
    uint32_t mk = 0;
    for (int ky = ylo; ky < yhi; ++ky) mk |= cols << (ky * a.kw);
    tmask = valid ? mk : 0u;
    poff = (a.proj.data && valid)
               ? (((n * a.proj.h + oy * a.proj_stride) * a.proj.w + ox * a.proj_stride) * (int)a.proj.pixel +
                  gd * (int)a.proj.gstride + xb)
               : (int)kOob;
  };
  tile_geometry();
  // Fetches K-block f_kb of tile f_tile into ring stage st.  Fetches past
  // the last tile read out-of-range offsets (zeros), so every call issues
  // the same loads.
  const auto rres = make_rsrc(a.res.data, a.res.data ? a.res.bytes : 0);
  auto fetch = [&](int st) __attribute__((always_inline)) {
    const bool live = f_tile < t_end;
    uint8_t *ws = lds + st * SST;
    if constexpr (RB == 2) {
      if (f_kb == 0) {  // the tile's shortcut codes, RPT 16-byte pieces per thread
        const int pt = f_it.pt;
        const int cbk = f_it.combo % ncb;
        const int gd = (f_it.combo / ncb + a.shuffle) % G;
        uint8_t *rb = lds + kStages * SST + ((f_tile - t_begin) & 1) * RSB;
#pragma unroll
        for (int i = 0; i < RPT; ++i) {
          const int c = tid + i * NT;
          const int m = pt * TM + c / (RPX / 16);
          const uint32_t ro = live && m < geo.M ? (uint32_t)((int64_t)m * a.res.pixel + gd * a.res.gstride + cbk * RPX +
                                                             (c % (RPX / 16)) * 16)
                                                : kOob;
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rres, (lds_ptr)(rb + i * NT * 16 + wave * 1024), 16, (int)ro, 0,
                                                   0, 0);
        }
      }
    }
#pragma unroll
    for (int i = 0; i < WLD; ++i) {
      const int c = tid + i * NT;  // piece of the K-block's weights
      const uint32_t woff = live ? wbase + (uint32_t)((c >> 7) * KB + f_kb) * kSlab + (c & 127) * 16 : kOob;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rw_src, (lds_ptr)(ws + i * NT * 16 + wave * 1024), 16, (int)woff, 0, 0,
                                               0);
    }
    if constexpr (STEM) {
#pragma unroll
      for (int i = 0; i < XLD; ++i) {
        const uint32_t xo = soff[i] >= 0 ? (uint32_t)(soff[i] + 2 * f_kb * rowb) : kOob;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rin, (lds_ptr)(ws + WST + i * NT * 16 + wave * 1024), 16, (int)xo, 0, 0,
                                                 0);
      }
    } else if (XALL || tid < XP) {
      uint32_t xo;
      __amdgpu_buffer_rsrc_t xr;
      if (f_kb < geo.kb_main) {
        xo = ((tmask >> f_tap) & 1u) ? (uint32_t)(off0 + f_tapoff + f_cblk * BLK) : kOob;
        xr = rin;
      } else {
        xo = (uint32_t)(poff + (f_kb - geo.kb_main) * BLK);
        xr = rpj;
      }
      __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_ptr)(ws + WST + wave * 1024), 16, (int)xo, 0, 0, 0);
    }
    if (++f_cblk == geo.cpb) {
      f_cblk = 0;
      ++f_tap;
      if (++f_kx == a.kw) { f_kx = 0; ++f_ky; }
      f_tapoff = f_ky * rowb + f_kx * pixb;
    }
    if (++f_kb == KB) {
      f_kb = f_tap = f_cblk = f_kx = f_ky = f_tapoff = 0;
      ++f_tile;
      tile_next(f_it, npt, ncb * G, nch);
      tile_geometry();
    }
  };

  // ---- compute side: tile c_tile, K-block c_kb
  int c_tile = t_begin, c_kb = 0;
  TileIt c_it = tile_at(t_begin, npt, ncb * G, nch);
  v16i acc[CB][PB];
  // Per tile, at its first K-block: zeroed accumulators.
  auto tile_start = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int cb = 0; cb < CB; ++cb)
#pragma unroll
      for (int pb = 0; pb < PB; ++pb)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[cb][pb][r] = 0;
  };
  auto tile_end = [&]() __attribute__((always_inline)) {
    const int pt = c_it.pt;
    const int cbk = c_it.combo % ncb;
    const int g = c_it.combo / ncb;
    const int gd = (g + a.shuffle) % G;
    uint32_t rw[CB][PB][2] = {};
    // this lane's shortcut codes: pixel block pb, channel block cb at
    // ra + pb 32 RPX + 8 cb
    const uint32_t ra = RB == 2 ? lds_base + kStages * SST + ((c_tile - t_begin) & 1) * RSB +
                                      (uint32_t)((wm * PB * 32 + l32) * RPX + wn * CB * 8)
                                : 0u;
    if constexpr (RB == 2) {
      uint2 r00, r01, r10, r11;  // r[pb][cb]
      asm volatile(
          "ds_read_b64 %0, %4\n\t"
          "ds_read_b64 %1, %4 offset:8\n\t"
          "ds_read_b64 %2, %4 offset:%5\n\t"
          "ds_read_b64 %3, %4 offset:%6\n\t"
          "s_waitcnt lgkmcnt(0)"
          : "=&v"(r00), "=&v"(r01), "=&v"(r10), "=&v"(r11)
          : "v"(ra), "i"(32 * RPX), "i"(32 * RPX + 8));
      rw[0][0][0] = r00.x; rw[0][0][1] = r00.y;
      rw[1][0][0] = r01.x; rw[1][0][1] = r01.y;
      rw[0][1][0] = r10.x; rw[0][1][1] = r10.y;
      rw[1][1][0] = r11.x; rw[1][1][1] = r11.y;
    }
    if constexpr (DUMP) {
      // accumulators of pixel mbase + 32 pb + l32, channels kc + 8 qi + 4 half + e
      const int64_t outC = (int64_t)G * a.cout, mbase = (int64_t)pt * TM + wm * PB * 32;
#pragma unroll
      for (int cb = 0; cb < CB; ++cb)
#pragma unroll
        for (int pb = 0; pb < PB; ++pb) {
          const int64_t mp = mbase + pb * 32 + l32;
          if (mp >= geo.M) continue;
          int32_t *dst = a.acc_dump + mp * outC + (int64_t)gd * a.cout + cbk * TN + wn * CB * 32 + cb * 32 + 4 * half;
#pragma unroll
          for (int qi = 0; qi < 4; ++qi) {
            v4i dv;
#pragma unroll
            for (int e = 0; e < 4; ++e) dv[e] = acc[cb][pb][4 * qi + e] >> (geo.scale == 16 ? 4 : 0);
            *(v4i *)(dst + 8 * qi) = dv;
          }
        }
    }
    const int rec = (c_it.combo == combo0 ? 0 : TN) + wn * CB * 32;  // first record of this wave's channels
    epilogue_fast_bo<2, CB, PB, RB, v16i>(
        a, geo, acc, rw, (int64_t)pt * TM + wm * PB * 32, g, gd, cbk * TN + wn * CB * 32, l32, half, rq_area + rec,
        rm_area + (RB ? rec : 0), ra, 32 * RPX);
  };
  // LDS addresses of this lane's operands in stage 0: activation half row
  // of pixel block 0, weight unit (j = 0) of channel block 0
  const uint32_t xaddr0 = lds_base + WST + (uint32_t)((wm * PB * 32 + l32) * BLK + half * (BLK / 2));
  const uint32_t aaddr0 = lds_base + (uint32_t)((wn * CB) * SLAB + (half * 32 + l32) * 16);
  // MFMA operands of one K-block: this lane's activation half rows of the two
  // pixel blocks and weight units a[j][cb], read by one asm statement that
  // also waits for them (early-clobber outputs: a result must not land in an
  // address register a later read of the statement still uses).
  struct OpsG { uint2 x0, x1; v4i a00, a01, a10, a11; };
  struct OpsS { v4i x0a, x0b, x1a, x1b, a00, a01, a10, a11; };  // stem: x[pb] words 0-3 / 4-7
  using Ops = typename std::conditional<STEM, OpsS, OpsG>::type;
  auto read_ops = [&](int stage, Ops &o) __attribute__((always_inline)) {
    const uint32_t xa = xaddr0 + stage * SST, aa = aaddr0 + stage * SST;
    if constexpr (STEM) {
      asm volatile(
          "ds_read_b128 %0, %8\n\t"
          "ds_read_b128 %1, %8 offset:16\n\t"
          "ds_read_b128 %2, %8 offset:2048\n\t"
          "ds_read_b128 %3, %8 offset:2064\n\t"
          "ds_read_b128 %4, %9\n\t"
          "ds_read_b128 %5, %9 offset:2048\n\t"
          "ds_read_b128 %6, %9 offset:1024\n\t"
          "ds_read_b128 %7, %9 offset:3072\n\t"
          "s_waitcnt lgkmcnt(0)"
          : "=&v"(o.x0a), "=&v"(o.x0b), "=&v"(o.x1a), "=&v"(o.x1b), "=&v"(o.a00), "=&v"(o.a01), "=&v"(o.a10),
            "=&v"(o.a11)
          : "v"(xa), "v"(aa));
      return;
    } else
    asm volatile(
        "ds_read_b64 %0, %6\n\t"
        "ds_read_b64 %1, %6 offset:512\n\t"
        "ds_read_b128 %2, %7\n\t"
        "ds_read_b128 %3, %7 offset:2048\n\t"
        "ds_read_b128 %4, %7 offset:1024\n\t"
        "ds_read_b128 %5, %7 offset:3072\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(o.x0), "=&v"(o.x1), "=&v"(o.a00), "=&v"(o.a01), "=&v"(o.a10), "=&v"(o.a11)
        : "v"(xa), "v"(aa));
  };
  auto mfmas = [&](const Ops &o) __attribute__((always_inline)) {
    if constexpr (STEM) {
      const v4i X[2][PB] = {{o.x0a, o.x1a}, {o.x0b, o.x1b}};
      const v4i A[2][CB] = {{o.a00, o.a01}, {o.a10, o.a11}};
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int pb = 0; pb < PB; ++pb)
#pragma unroll
          for (int cb = 0; cb < CB; ++cb)
            acc[cb][pb] = __builtin_amdgcn_mfma_i32_32x32x32_i8(A[j][cb], X[j][pb], acc[cb][pb], 0, 0, 0);
      return;
    } else {
    Raw xr[PB];
    xr[0].w[0] = o.x0.x; xr[0].w[1] = o.x0.y;
    xr[1].w[0] = o.x1.x; xr[1].w[1] = o.x1.y;
    const v4i A[2][CB] = {{o.a00, o.a01}, {o.a10, o.a11}};
#pragma unroll
    for (int j = 0; j < 2; ++j) {
#pragma unroll
      for (int pb = 0; pb < PB; ++pb) {
        const v4i bop = act_operand<B>(xr[pb], j);
#pragma unroll
        for (int cb = 0; cb < CB; ++cb)
          acc[cb][pb] = __builtin_amdgcn_mfma_i32_32x32x32_i8(A[j][cb], bop, acc[cb][pb], 0, 0, 0);
      }
    }
    }
  };
  // K-block gk: wait until this wave's loads of it have landed, barrier
  // (everyone's have, and everyone is done with the previous stage, which
  // the next fetch reuses), fetch the K-block kStages - 1 ahead, then read
  // the operands, run the MFMAs, and finish the tile after its last
  // K-block.  A tile's shortcut codes (two buffers) are safe while
  // kb_total >= kStages.
  for (int st = 0; st < kStages - 1; ++st) fetch(st);
  for (int gk = 0; gk < total; ++gk) {
    const int st = gk % kStages;
    __builtin_amdgcn_s_waitcnt(waitcnt_vm((kStages - 2) * LPK));
    ring_barrier();
    fetch((st + kStages - 1) % kStages);
    if (c_kb == 0) tile_start();
    Ops o;
    read_ops(st, o);
    __builtin_amdgcn_sched_barrier(0);
    mfmas(o);
    if (++c_kb == KB) {
      tile_end();
      c_kb = 0;
      ++c_tile;
      tile_next(c_it, npt, ncb * G, nch);
    }
  }
}

// ---------------------------------------------------------------- stem + max pool
// The 8-bit stem followed by the 3x3 / stride 2 / pad 1 max pool, fused: the
// max pool is taken over the stem's int32 accumulators and only the pooled
// values are requantised.  Exact: the requant q = clamp(floor((t M +
// 2^(sh-1)) / 2^sh), 0, 2^b - 1) is non-decreasing in t for M >= 0 (the
// fast epilogue, which this kernel has, requires that), so the max of the
// requantised values equals the requant of the max.
//
// The stem is a 7x7 / stride 2 filter over 4-byte pixels (3 channels and a
// zero byte) with an explicit zero border.  Its K is laid out as one 32-byte
// K-step per filter row (8 taps x 4 bytes, tap 7 and the fourth byte with
// zero weight): 7 K-steps, 224 of which 147 are real.  Lane half h of an
// MFMA operand holds taps 4h .. 4h + 3 of the row, which for output column c
// are the 16 contiguous input bytes 8c + 16h ..: the operand is read straight
// out of the staged input row, so the activations are staged once per
// output row (its 7 input rows) instead of once per K-step and pixel.  Each
// row is staged twice, the second copy 8 bytes on, so that odd columns
// (8 mod 16 bytes) also read 16-byte aligned operands.  The weights of a
// wave's 64 channels (7 x 2 K-steps of 16 bytes a lane) stay in registers.
//
// A step is one output row (wo <= 125 columns) of one image and 128 output
// channels, 2 x 2 waves of 2 x 2 32 x 32 blocks (wave (wn, wm): channels
// 64 wn .. + 63).  Column halves overlap by one column: wm = 0 holds columns
// 0 .. 63, wm = 1 columns 63 .. 126, lane l of pixel block pb column
// 63 wm + 2 l + pb.  Pooled column 32 wm + l then needs the lane's two
// columns and one of its neighbour lane (l - 1 for wm = 0, l + 1 for
// wm = 1), a DPP shift within the wave.  Work units are pooled rows (image,
// channel block, k); a unit takes output rows 2k and 2k + 1, and pooled row
// k also needs row 2k - 1, which the previous unit of the same run left in
// registers (a run starting inside an image recomputes it).
namespace sp {
constexpr int NT = 256;
constexpr int KH = 7;                // filter rows = K-steps
constexpr int RB = 1024;             // LDS bytes of one staged copy of an input row
constexpr int SET = 8 * 2 * RB;      // an output row's input rows 0 .. 7, two copies each
constexpr int kSets = 3;             // ring of staged output rows, two ahead of the MFMAs

// Row steps of a run: phase 0 recomputes row 2k - 1, 1 is row 2k, 2 row 2k + 1.
struct RowIt {
  int u, phase;
};
__device__ __forceinline__ RowIt row_first(int u, int ho2) { return {u, (u % ho2) > 0 ? 0 : 1}; }
__device__ __forceinline__ void row_next(RowIt &it, int ho, int ho2) {
  if (it.phase == 0) { it.phase = 1; return; }
  if (it.phase == 1 && 2 * (it.u % ho2) + 1 < ho) { it.phase = 2; return; }
  ++it.u;
  it.phase = 1;
}
__device__ __forceinline__ int row_of(const RowIt &it, int ho2) {
  const int k = it.u % ho2;
  return it.phase == 0 ? 2 * k - 1 : 2 * k + (it.phase - 1);
}
}  // namespace sp

// Stem weights by filter row: [cout / 32][KH][half][ch][16 B], lane (half,
// ch) of K-step r holding taps 4 half .. + 3 of row r for channel ch, the
// input's padding byte and taps past kw masked to zero.  One thread per
// 16-byte lane operand.
__global__ void prepack_stem_rows_kernel(ConvArgs a, uint8_t *wp) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= (int64_t)a.cout * sp::KH * 2) return;
  const int lane = (int)(t & 63), r = (int)((t >> 6) % sp::KH);
  const int k = (int)(t / (64 * sp::KH)) * 32 + (lane & 31), h = lane >> 5;
  const uint32_t *wr = (const uint32_t *)(a.w + ((int64_t)k * a.kh + r) * a.kw * 4);
  const uint32_t cmask = a.in.cpg >= 4 ? 0xffffffffu : ((1u << (8 * a.in.cpg)) - 1u);
  uint32_t o[4];
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    const int kx = 4 * h + d;
    o[d] = kx < a.kw ? (wr[kx] & cmask) : 0u;
  }
  *(uint4 *)(wp + t * 16) = make_uint4(o[0], o[1], o[2], o[3]);
}

// Runs hold at most ho2 units (the launcher's grid), so a run meets at most
// two channel blocks, cbb0 and cbb0 + 1 (mod ncb): their requant constants
// sit in LDS.
__global__ __launch_bounds__(sp::NT, 2) void stem_pool_kernel(ConvArgs a, Geo geo, ActView po, const uint8_t *wrow,
                                                              int units) {
  using namespace sp;
  __shared__ __attribute__((aligned(1024))) uint8_t lds[kSets * SET];
  __shared__ RqConst rq_area[256];
  if (needs_general(a, geo, 0)) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, half = lane >> 5;
  const int wn = wave >> 1, wm = wave & 1;
  const int ho = a.ho, wo = a.wo, ho2 = po.h, wo2 = po.w;
  const int ncb = a.cout / 128;
  // balanced runs of units per XCD (as the tiled kernel's tiles)
  const int P = (int)gridDim.x >> 3;
  const int x = (int)(blockIdx.x & 7), y = (int)(blockIdx.x >> 3);
  const int Tq = units >> 3, Tr = units & 7;
  const int Tx = Tq + (x < Tr ? 1 : 0);
  const int base = Tx / P, ex = Tx % P;
  const int u_begin = x * Tq + min(x, Tr) + y * base + min(y, ex);
  const int u_end = u_begin + base + (y < ex ? 1 : 0);
  if (u_begin >= u_end) return;  // no barrier yet
  const int cbb0 = (u_begin / ho2) % ncb;
  for (int c = tid; c < 256; c += NT) rq_area[c] = geo.rq[(c < 128 ? cbb0 : (cbb0 + 1) % ncb) * 128 + (c & 127)];
  __syncthreads();
  const uint32_t lds_base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t *)lds;
  typedef __attribute__((address_space(3))) void *lds_ptr;
  const auto rin = make_rsrc(a.in.data, a.in.bytes);
  const auto rout = make_rsrc(po.data, po.bytes);
  const int rowb = a.in.w * (int)a.in.pixel;  // <= RB (launcher)

  // ---- fetcher: output row f_it.  Wave w stages input rows w and w + 4 of
  // the row's window (row 7 is never read: no filter row 7); copy 1 of a row
  // starts 8 bytes on.  Lanes past the row's end load the next row's first
  // bytes (or zeros past the tensor), which no operand reads.
  RowIt f_it = row_first(u_begin, ho2);
  int f_set = 0;
  auto fetch = [&]() __attribute__((always_inline)) {
    const bool live = f_it.u < u_end;
    const int n = f_it.u / (ho2 * ncb);
    const uint32_t rbase = live ? (uint32_t)((n * a.in.h + 2 * row_of(f_it, ho2) + wave) * rowb + lane * 16) : kOob;
    uint8_t *ws = lds + f_set * SET + wave * 2 * RB;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int cp = 0; cp < 2; ++cp)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rin, (lds_ptr)(ws + (8 * i + cp) * RB), 16,
                                                 (int)(rbase + (uint32_t)(4 * i * rowb + 8 * cp)), 0, 0, 0);
    if (live) row_next(f_it, ho, ho2);
    f_set = f_set == kSets - 1 ? 0 : f_set + 1;
  };

  // ---- compute side
  RowIt c_it = row_first(u_begin, ho2);
  int c_set = 0, w_cbb = -1;
  v16i acc[2][2];     // [cb][pb]
  int32_t st[2][16];  // per cb: row 2k - 1 pooled across columns, or the running max of rows 2k - 1, 2k
  v4i W[KH][2];       // [K-step][cb]
  // operand address of pixel block pb: column c (slots past the last column
  // read the last column again: the window of a pooled column reaching past
  // the row holds the last column, so the duplicate leaves the max unchanged)
  uint32_t xa[2];
#pragma unroll
  for (int pb = 0; pb < 2; ++pb) {
    const int c = min(63 * wm + 2 * l32 + pb, wo - 1);
    xa[pb] = lds_base + (uint32_t)((c & 1) * RB + 16 * (c >> 1) + 16 * half);
  }
  // the lanes whose pooling neighbour is missing from the DPP shift: the
  // wave's end lane (no source lane) and the lane whose source lies in the
  // other lane half (column -1 for wm = 0, column 127 for wm = 1)
  const bool half_edge = wm ? l32 == 31 : l32 == 0;
  // pooled column px = 32 wm + l; its byte offset in a pooled row plus this
  // lane's word of the wave's channels (word 2 (4 cbb + 2 wn + cb) + half)
  const int px = 32 * wm + l32;
  int out_lane = px * (int)po.pixel + (wn * 4 + half) * 4;
  asm volatile("" : "+v"(out_lane));  // kept as one 32-bit register
  auto finish_row = [&]() __attribute__((always_inline)) {
    const int k = c_it.u % ho2;
    const int cbb = (c_it.u / ho2) % ncb, n = c_it.u / (ho2 * ncb);
    // columns 2p - 1 .. 2p + 1 of pooled column p = 32 wm + l: the lane's
    // two columns and column 2p - 1 from lane l - 1 (wm = 0) or 2p + 1 from
    // lane l + 1 (wm = 1); then the rows.  st: row 2k - 1 (pooled across
    // columns) before row 2k, the max of rows 2k - 1 and 2k before row
    // 2k + 1; after the last row of pooled row k it holds that row, which is
    // requantised; row 2k + 1, kept in nx, then becomes st for row k + 1.
    int32_t nx[2][16];
    auto pool_row = [&](auto WMC) __attribute__((always_inline)) {
      constexpr int WMV = decltype(WMC)::value;
      // neighbour column by a DPP wave shift folded into the max (lane i
      // reads lane i - 1 for wm = 0, i + 1 for wm = 1; the end lane, which
      // has no source, reads zero); the edge lanes (that end lane and the
      // lane whose neighbour lies in the other lane half) take their own
      // column instead (a duplicate leaves the max unchanged)
      auto hmax = [&](int cb, int i) __attribute__((always_inline)) {
        const int32_t v0 = acc[cb][0][i], v1 = acc[cb][1][i];
        int32_t t;
        if constexpr (WMV == 0) {
          t = max(__builtin_amdgcn_update_dpp(0, v1, 0x138 /* wave_shr:1 */, 0xf, 0xf, true), v0);
          t = half_edge ? v0 : t;
          return max(t, v1);
        } else {
          t = max(__builtin_amdgcn_update_dpp(0, v0, 0x130 /* wave_shl:1 */, 0xf, 0xf, true), v1);
          t = half_edge ? v1 : t;
          return max(t, v0);
        }
      };
      if (c_it.phase == 2) {
#pragma unroll
        for (int cb = 0; cb < 2; ++cb)
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            nx[cb][i] = hmax(cb, i);
            st[cb][i] = max(st[cb][i], nx[cb][i]);
          }
      } else if (c_it.phase == 1 && k > 0) {
#pragma unroll
        for (int cb = 0; cb < 2; ++cb)
#pragma unroll
          for (int i = 0; i < 16; ++i) st[cb][i] = max(st[cb][i], hmax(cb, i));
      } else {
#pragma unroll
        for (int cb = 0; cb < 2; ++cb)
#pragma unroll
          for (int i = 0; i < 16; ++i) st[cb][i] = hmax(cb, i);
      }
    };
    if (wm == 0) pool_row(std::integral_constant<int, 0>{});
    else pool_row(std::integral_constant<int, 1>{});
    if (c_it.phase == 0 || (c_it.phase == 1 && 2 * k + 1 < ho)) return;
    // requant the pooled row and store it: channel 128 cbb + 64 wn + 32 cb + 8 qi + 4 half + e
    const int orow = ((n * ho2 + k) * wo2) * (int)po.pixel;
    const RqConst *rq = rq_area + (cbb == cbb0 ? 0 : 128) + wn * 64;
    // the constants of quad j + 1 are read while quad j is requantised (two
    // quads' constants in registers, which the dead accumulators free)
    RqConst qc[2][4];
    auto load_quad = [&](int j) __attribute__((always_inline)) {
      const int cq = (j >> 2) * 32 + 8 * (j & 3) + 4 * half;
#pragma unroll
      for (int e = 0; e < 4; ++e) qc[j & 1][e] = rq[cq + e];
    };
    load_quad(0);
#pragma unroll
    for (int cb = 0; cb < 2; ++cb) {
      uint32_t qv[4];
#pragma unroll
      for (int qi = 0; qi < 4; ++qi) {
        const int j = 4 * cb + qi;
        __builtin_amdgcn_sched_barrier(0);
        if (j < 7) load_quad(j + 1);
        __builtin_amdgcn_sched_barrier(0);
        uint32_t qword = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const double d = __builtin_fma((double)st[cb][4 * qi + e], qc[j & 1][e].s, qc[j & 1][e].o);
          uint32_t q;
          asm("v_cvt_u32_f64 %0, %1" : "=v"(q) : "v"(d));
          qword |= min(q, 3u) << (2 * e);
        }
        qv[qi] = qword;
      }
      const auto p0 = __builtin_amdgcn_permlane32_swap(qv[0], qv[2], false, false);  // as in epilogue_fast_bo
      const auto p1 = __builtin_amdgcn_permlane32_swap(qv[1], qv[3], false, false);
      const uint32_t Q[4] = {p0[0], p0[1], p1[0], p1[1]};
      if (px < wo2)
        __builtin_amdgcn_raw_buffer_store_b32(Q[0] | (Q[1] << 8) | (Q[2] << 16) | (Q[3] << 24), rout,
                                              out_lane + cbb * 32 + cb * 8, orow, 0);
    }
    if (c_it.phase == 2) {
#pragma unroll
      for (int cb = 0; cb < 2; ++cb)
#pragma unroll
        for (int i = 0; i < 16; ++i) st[cb][i] = nx[cb][i];
    }
  };

  int rows = 0;
  for (RowIt it = row_first(u_begin, ho2); it.u < u_end; row_next(it, ho, ho2)) ++rows;
  fetch();
  fetch();
  for (int gk = 0; gk < rows; ++gk) {
    // the wave's weights, loaded when the channel block changes (at most
    // twice a run)
    const int cbb = (c_it.u / ho2) % ncb;
    if (cbb != w_cbb) {
      w_cbb = cbb;
      const uint8_t *wsrc = wrow + ((int64_t)(cbb * 4 + 2 * wn) * KH * 64 + lane) * 16;
#pragma unroll
      for (int cb = 0; cb < 2; ++cb)
#pragma unroll
        for (int r = 0; r < KH; ++r) W[r][cb] = *(const v4i *)(wsrc + (cb * KH + r) * 1024);
      __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));  // here, not inside every later row's MFMAs
    }
#pragma unroll
    for (int cb = 0; cb < 2; ++cb)
#pragma unroll
      for (int pb = 0; pb < 2; ++pb)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[cb][pb][r] = 0;
    // this row's rows staged (each wave its own four loads; one row ahead
    // stays in flight), then visible to every wave, and the set of the row
    // before free for the row two ahead
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(4));
    ring_barrier();
    fetch();
    const uint32_t so = (uint32_t)(c_set * SET);
    const uint32_t x0 = xa[0] + so, x1 = xa[1] + so;
    v4i X[KH][2];
    asm volatile(
        "ds_read_b128 %0, %8\n\t"
        "ds_read_b128 %1, %9\n\t"
        "ds_read_b128 %2, %8 offset:2048\n\t"
        "ds_read_b128 %3, %9 offset:2048\n\t"
        "ds_read_b128 %4, %8 offset:4096\n\t"
        "ds_read_b128 %5, %9 offset:4096\n\t"
        "ds_read_b128 %6, %8 offset:6144\n\t"
        "ds_read_b128 %7, %9 offset:6144"
        : "=&v"(X[0][0]), "=&v"(X[0][1]), "=&v"(X[1][0]), "=&v"(X[1][1]), "=&v"(X[2][0]), "=&v"(X[2][1]),
          "=&v"(X[3][0]), "=&v"(X[3][1])
        : "v"(x0), "v"(x1));
    asm volatile(
        "ds_read_b128 %0, %6 offset:8192\n\t"
        "ds_read_b128 %1, %7 offset:8192\n\t"
        "ds_read_b128 %2, %6 offset:10240\n\t"
        "ds_read_b128 %3, %7 offset:10240\n\t"
        "ds_read_b128 %4, %6 offset:12288\n\t"
        "ds_read_b128 %5, %7 offset:12288"
        : "=&v"(X[4][0]), "=&v"(X[4][1]), "=&v"(X[5][0]), "=&v"(X[5][1]), "=&v"(X[6][0]), "=&v"(X[6][1])
        : "v"(x0), "v"(x1));
    // the first eight reads have landed (LDS reads complete in order)
    asm volatile("s_waitcnt lgkmcnt(6)"
                 : "+v"(X[0][0]), "+v"(X[0][1]), "+v"(X[1][0]), "+v"(X[1][1]), "+v"(X[2][0]), "+v"(X[2][1]),
                   "+v"(X[3][0]), "+v"(X[3][1]));
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int pb = 0; pb < 2; ++pb)
#pragma unroll
        for (int cb = 0; cb < 2; ++cb)
          acc[cb][pb] = __builtin_amdgcn_mfma_i32_32x32x32_i8(W[r][cb], X[r][pb], acc[cb][pb], 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);  // the rows 0 - 3 MFMAs issue before the last reads are awaited
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(X[4][0]), "+v"(X[4][1]), "+v"(X[5][0]), "+v"(X[5][1]), "+v"(X[6][0]), "+v"(X[6][1]));
#pragma unroll
    for (int r = 4; r < KH; ++r)
#pragma unroll
      for (int pb = 0; pb < 2; ++pb)
#pragma unroll
        for (int cb = 0; cb < 2; ++cb)
          acc[cb][pb] = __builtin_amdgcn_mfma_i32_32x32x32_i8(W[r][cb], X[r][pb], acc[cb][pb], 0, 0, 0);
    finish_row();
    row_next(c_it, ho, ho2);
    c_set = c_set == kSets - 1 ? 0 : c_set + 1;
  }
  // no staging load may land after the workgroup's LDS is released
  __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
}

// ---------------------------------------------------------------- FP4 grouped kernel
// 2-bit grouped layers on the FP4 (E2M1) matrix cores, one workgroup per
// tile.  A tile is TN = WN CB 32 output channels x TM = WM PB 32 output
// pixels of one group; wave (wn, wm) owns CB x PB blocks of 32 x 32.  Per
// 64-code K-block the workgroup stages TN / 32 FP4 weight slabs (1 KB each,
// prepack_fp4_kernel) and the TM pixels' packed codes (16 bytes each) in a
// ring of S LDS stages with buffer_load ... lds, S - 1 K-blocks ahead of the
// MFMAs (one barrier per K-block).  Per K-block a lane's fetch offsets change
// only through the scalar offset (K-block within the tap, weight slab step);
// the per-lane activation offset and its in-image test are redone when the
// tap changes.  The K-blocks of a fused projection follow the main ones.
// Tiles are dealt in XCD-contiguous runs (workgroup i runs on XCD i mod 8),
// in the chunked order of tile_at, so an XCD's L2 holds the input lines its
// in-flight tiles share.  Epilogue: epilogue_fast_bo (fp64-exact requant);
// a layer whose requant needs the int64 path leaves at once (its general
// partner runs instead).  DUMP: also write the int32 accumulators.
// A value the compiler is told is the same in every lane of the wave.
__device__ __forceinline__ int uniform_int(int v) { return __builtin_amdgcn_readfirstlane(v); }

namespace f4 {
template <int CB, int PB, int WN, int WM, int B = 2>
struct Cfg {
  static constexpr int NT = WN * WM * 64;
  static constexpr int TN = WN * CB * 32, TM = WM * PB * 32;
  static constexpr int SLAB = B == 2 ? kSlab4 : kSlab6;  // weight bytes per 32 channels and K-block
  static constexpr int PPX = B == 2 ? 1 : 2;             // 16-byte activation pieces per pixel and K-block
  static constexpr int WST = TN / 32 * SLAB;  // weight bytes of a K-block
  static constexpr int XST = TM * 16 * PPX;   // activation bytes of a K-block
  static constexpr int SST = WST + XST;
  static constexpr int WP = WST / 16, XP = XST / 16;  // 16-byte pieces
  static_assert(WP % 64 == 0 && XP % 64 == 0 && WP <= 2 * NT && XP <= 2 * NT, "whole waves of pieces");
  static constexpr int WL = WP > NT ? 2 : 1, XL = XP > NT ? 2 : 1;  // loads per loading thread
  // whether wave w issues weight (activation) load i: fewer pieces than
  // threads go to the last (first) waves, more to every thread and then to
  // the first waves
  static constexpr bool wloads(int w, int i) { return WP < NT ? (i == 0 && 64 * w >= NT - WP) : 64 * w + i * NT < WP; }
  static constexpr bool xloads(int w, int i) { return XP < NT ? (i == 0 && 64 * w < XP) : 64 * w + i * NT < XP; }
  static constexpr int loads(int w) {
    int n = 0;
    for (int i = 0; i < WL; ++i) n += wloads(w, i) ? 1 : 0;
    for (int i = 0; i < XL; ++i) n += xloads(w, i) ? 1 : 0;
    return n;
  }
  static constexpr int min_loads() {
    int m = 1 << 30;
    for (int w = 0; w < NT / 64; ++w) m = loads(w) < m ? loads(w) : m;
    return m;
  }
  // loads per K-block of the waves with the fewest (the ring waits on that)
  static constexpr int LPK = min_loads();
  static_assert(LPK >= 1, "every wave loads in every K-block");
  static constexpr int RPX = TN / 4;          // shortcut code bytes per pixel
  static constexpr int RSB = TM * RPX;        // shortcut codes of a tile
};
}  // namespace f4

// B = 2: FP4 operands (conv_fp4_kernel); B = 3: 3-bit layers on FP6 (E2M3)
// matrix cores (conv_fp6_kernel): 1536-byte weight slabs (prepack_fp6_kernel),
// each pixel's K-block staged as its two 12-byte chunks in 16-byte pieces
// (the chunk's three words at the start of each), fp6_operand, and a 3-bit
// fast epilogue; no shortcut.
// F32 (B = 2): the fp32 requant of requant_prep_f32_kernel; K-block 0's
// MFMAs start from the channels' bias / 4 instead of zero.
// KS = 2 (B = 2, for layers with few tiles): the workgroup is two groups of
// WN x WM waves; a ring stage holds two consecutive K-blocks (the same tap:
// the host takes this build only for an even K-block count per tap and an
// even projection), group h fetching and multiplying K-block 2 s + h of
// stage s; at the end group 1 adds its accumulators to group 0's through
// LDS (the two partial sums are exact, so is their sum) and group 0 runs
// the epilogue.  Twice the waves per tile, half the K loop each.
template <int CB, int PB, int WN, int WM, int RB, bool DUMP, int S, int B, bool F32 = false, int KS = 1>
__device__ __forceinline__ void conv_fpx_tile(const ConvArgs &a, const Geo &geo, int npt, int ncb, int nch) {
  using C = f4::Cfg<CB, PB, WN, WM, B>;
  // NT: the threads of one group; SSB: one K-block of a stage; SST: a stage
  constexpr int NT = C::NT, TN = C::TN, TM = C::TM, WST = C::WST, SSB = C::SST, SST = KS * SSB;
  static_assert(KS == 1 || (KS == 2 && B == 2 && PB == 2), "the K split takes FP4 layers with 2 x 2 blocks");
  // the K split's reduction buffer: group 0's waves x 16 chunks x 64 lanes x 16 bytes, over the ring
  constexpr int RED = KS == 2 ? (NT / 64) * 16 * 64 * 16 : 0;
  constexpr int RING = S * SST > RED ? S * SST : RED;
  constexpr int RPT = RB ? C::RSB / (NT * 16) : 0;  // 16-byte shortcut pieces per thread
  static_assert(RB == 0 || RPT * NT * 16 == C::RSB, "whole shortcut pieces per thread");
  static_assert(CB == 2 && (PB == 2 || PB == 4), "operand reads are written for 2 x 2 and 2 x 4 blocks");
  static_assert(B == 2 || (B == 3 && PB == 2 && RB == 0), "FP6: 2 x 2 blocks, no shortcut");
  static_assert(!F32 || B == 2, "the fp32 requant takes FP4 accumulators");
  constexpr int XB = B == 2 ? 16 : 24;  // activation bytes of a pixel's K-block
  __shared__ __attribute__((aligned(1024))) uint8_t lds[RING + (RB ? C::RSB : 16)];
  __shared__ RqConst rq_area[TN];
  __shared__ int32_t rm_area[RB ? TN : 1];

  // the launcher takes 2-bit outputs and 2-bit (or no) shortcuts only; a
  // layer whose fp64 requant could be inexact runs on the general partner
  if (int64_flag(a, geo) || a.out.bits != B || RB < 0) return;
  const int G = a.in.groups;
  const int T = npt * ncb * G;
  // workgroup i -> XCD x = i mod 8, which takes the x-th eighth of the tiles
  const int x8 = (int)(blockIdx.x & 7), j = (int)(blockIdx.x >> 3);
  const int Tq = T >> 3, Tr = T & 7;
  if (j >= Tq + (x8 < Tr ? 1 : 0)) return;  // no barrier yet
  const int t = x8 * Tq + min(x8, Tr) + j;
  const TileIt it = tile_at(t, npt, ncb * G, nch);
  const int pt = it.pt, cbk = it.combo % ncb, g = it.combo / ncb;
  const int gd = (g + a.shuffle) % G;
  // tid, wave: within the thread's group kh (KS = 2: of the two)
  const int kh = KS == 2 ? uniform_int((int)threadIdx.x / NT) : 0;
  const int tid = (int)threadIdx.x - kh * NT, lane = tid & 63;
  const int wave = uniform_int(tid >> 6);  // LDS destinations in scalar registers
  const int l32 = lane & 31, half = lane >> 5;
  const int wn = wave / WM, wm = wave % WM;
  const int KB = geo.kb_total, KM = geo.kb_main;

  // requant constants (and shortcut multipliers) of the tile's TN channels;
  // F32: the fp32 scales, then bias / 4, in rq_area's bytes, and the
  // shortcut scales res_mult / 4 as fp32 bits in rm_area
  const int64_t ch0 = (int64_t)g * a.cout + cbk * TN;
  float *const sc_area = (float *)rq_area, *const b4_area = sc_area + TN;
  for (int c = (int)threadIdx.x; c < TN; c += NT * KS) {
    if constexpr (F32) {
      const int64_t nall = (int64_t)G * a.cout;
      const float *f32c = (const float *)(geo.rq + nall + 1);
      sc_area[c] = f32c[ch0 + c];
      b4_area[c] = f32c[nall + ch0 + c];
      if constexpr (RB != 0) rm_area[c] = __builtin_bit_cast(int32_t, f32c[2 * nall + ch0 + c]);
    } else {
      rq_area[c] = geo.rq[ch0 + c];
      if constexpr (RB != 0) rm_area[c] = a.res_mult[ch0 + c];
    }
  }
  typedef __attribute__((address_space(3))) void *lds_ptr;
  const uint32_t lds_base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t *)lds;

  const auto rw_src = make_rsrc(geo.wp, (int64_t)G * a.cout * KB * (C::SLAB / 32));
  const auto rin = make_rsrc(a.in.data, a.in.bytes);
  const auto rpj = a.proj.data ? make_rsrc(a.proj.data, a.proj.bytes)
                               : make_rsrc(a.in.data, 0);
  const auto rres = make_rsrc(a.res.data, a.res.data ? a.res.bytes : 0);
  const int pixb = (int)a.in.pixel, rowb = a.in.w * pixb;

  // ---- this thread's fetch pieces (wave w issues load i if C::wloads /
  // C::xloads (w, i)).  Weights: piece c = tid - (NT - WP) (or tid + i NT)
  // of the tile's slabs: slab c / (SLAB / 16), 16-byte piece c % (SLAB / 16).
  // Activations, piece q = tid + i NT: B = 2, pixel q of the tile; B = 3,
  // chunk (q >> 5) & 1 of pixel 32 (q >> 6) + (q & 31).
  constexpr int PPS = C::SLAB / 16;  // pieces per slab
  const int wc = C::WP >= NT ? tid : tid - (NT - C::WP);
  uint32_t woff[C::WL];
#pragma unroll
  for (int i = 0; i < C::WL; ++i) {
    const int c = wc + i * NT;
    woff[i] = (uint32_t)((((int64_t)g * (a.cout / 32) + cbk * (TN / 32) + c / PPS) * KB) * C::SLAB + (c % PPS) * 16);
  }
  const int HW = a.ho * a.wo;
  const float inv_hw = geo.inv_hw, inv_wo = geo.inv_wo;
  int off0[C::XL], poff[C::XL];
  uint32_t tmask[C::XL];
#pragma unroll
  for (int i = 0; i < C::XL; ++i) {
    const int q = tid + i * NT;
    const int m = pt * TM + (B == 2 ? q : 32 * (q >> 6) + (q & 31));
    const bool valid = m < geo.M;
    const int mm = valid ? m : 0;
    const int n = fdiv(mm, HW, inv_hw);
    const int rem = mm - n * HW;
    const int oy = fdiv(rem, a.wo, inv_wo);
    const int ox = rem - oy * a.wo;
    const int iy0 = oy * a.stride - a.pad, ix0 = ox * a.stride - a.pad;
    off0[i] = ((n * a.in.h + iy0) * a.in.w + ix0) * pixb + g * (int)a.in.gstride + (B == 3 ? 12 * ((q >> 5) & 1) : 0);
    const int xlo = max(0, -ix0), xhi = min(a.kw, a.in.w - ix0);
    const uint32_t below = xhi >= 32 ? 0xffffffffu : ((1u << max(xhi, 0)) - 1u);
    const uint32_t cols = xhi > xlo ? (below & ~((1u << xlo) - 1u)) : 0u;
    const int ylo = max(0, -iy0), yhi = min(a.kh, a.in.h - iy0);
    uint32_t mk = 0;
    for (int ky = ylo; ky < yhi; ++ky) mk |= cols << (ky * a.kw);
    tmask[i] = valid ? mk : 0u;
    poff[i] = (a.proj.data && valid)
                  ? (((n * a.proj.h + oy * a.proj_stride) * a.proj.w + ox * a.proj_stride) * (int)a.proj.pixel +
                     gd * (int)a.proj.gstride)
                  : (int)kOob;
  }
  // fetch cursor: K-block f_kb = tap f_tap, block f_c of it; vo: the
  // activation pieces' offsets for the current tap (kOob if outside)
  int f_kb = 0, f_c = 0, f_tap = 0, f_kx = 0, f_tapoff = 0;
  uint32_t vo[C::XL];
  auto tap_offsets = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < C::XL; ++i) vo[i] = ((tmask[i] >> f_tap) & 1u) ? (uint32_t)(off0[i] + f_tapoff) : kOob;
  };
  tap_offsets();
  auto fetch = [&](int st) __attribute__((always_inline)) {
    uint8_t *ws = lds + st * SST + kh * SSB;  // this group's K-block f_kb + kh of the stage
    if constexpr (RB == 2) {
      if (f_kb == 0 && kh == 0) {  // the tile's shortcut codes, RPT pieces per thread (before K-block 0's loads)
#pragma unroll
        for (int i = 0; i < RPT; ++i) {
          const int c = tid + i * NT;
          const int m = pt * TM + c / (C::RPX / 16);
          const uint32_t ro = m < geo.M ? (uint32_t)((int64_t)m * a.res.pixel + gd * a.res.gstride + cbk * C::RPX +
                                                     (c % (C::RPX / 16)) * 16)
                                        : kOob;
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rres, (lds_ptr)(lds + RING + i * NT * 16 + wave * 1024), 16,
                                                   (int)ro, 0, 0, 0);
        }
      }
    }
#pragma unroll
    for (int i = 0; i < C::WL; ++i)
      if (C::wloads(wave, i))
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rw_src, (lds_ptr)(ws + ((wc + i * NT) & ~63) * 16), 16, (int)woff[i],
                                                 (f_kb + kh) * C::SLAB, 0, 0);
    if (f_kb < KM) {
#pragma unroll
      for (int i = 0; i < C::XL; ++i)
        if (C::xloads(wave, i))
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rin, (lds_ptr)(ws + WST + i * NT * 16 + wave * 1024), 16, (int)vo[i],
                                                   (f_c + kh) * XB, 0, 0);
    } else {
#pragma unroll
      for (int i = 0; i < C::XL; ++i)
        if (C::xloads(wave, i))
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rpj, (lds_ptr)(ws + WST + i * NT * 16 + wave * 1024), 16,
                                                   (int)poff[i], (f_kb + kh - KM) * 16, 0, 0);
    }
    f_kb += KS;
    f_c += KS;
    if (f_c == geo.cpb) {  // next tap
      f_c = 0;
      ++f_tap;
      f_tapoff += pixb;
      if (++f_kx == a.kw) {
        f_kx = 0;
        f_tapoff += rowb - a.kw * pixb;
      }
      tap_offsets();
    }
  };

  // ---- compute side (K-block 0's MFMAs take a zero C operand, or F32 the
  // channels' bias / 4, so the accumulators need no initialisation)
  v16f acc[CB][PB];
  v16f c0[CB];  // F32: K-block 0's C operand of channel block cb
  // LDS addresses of this lane's operands in stage 0: activation half row of
  // pixel block 0 (blocks 512 bytes apart), weight unit of channel block 0
  // (blocks 1 KB apart)
  // (B = 3: chunk half of pixel block 0 at 1 KB blocks, the weight unit's
  // first 16 bytes and its last 8 bytes, slabs 1536 bytes apart)
  // (KS = 2: in this group's half of the stage)
  const uint32_t gbase = lds_base + (uint32_t)(kh * SSB);
  const uint32_t xaddr0 = gbase + WST +
                          (uint32_t)(B == 2 ? (wm * PB * 32 + l32) * 16 + half * 8 : ((wm * PB) * 64 + lane) * 16);
  const uint32_t aaddr0 = gbase + (uint32_t)((wn * CB) * C::SLAB + lane * 16);
  const uint32_t baddr0 = gbase + (uint32_t)((wn * CB) * C::SLAB + 1024 + lane * 8);
  auto kblock = [&](int st, bool first) __attribute__((always_inline)) {
    const uint32_t xa = xaddr0 + st * SST, aa = aaddr0 + st * SST;
    if constexpr (B == 3) {
      const uint32_t ba = baddr0 + st * SST;
      v4i x0, x1, A0, A1;
      v2i B0, B1;
      asm volatile(
          "ds_read_b128 %0, %6\n\t"
          "ds_read_b128 %1, %6 offset:1024\n\t"
          "ds_read_b128 %2, %7\n\t"
          "ds_read_b64 %3, %8\n\t"
          "ds_read_b128 %4, %7 offset:1536\n\t"
          "ds_read_b64 %5, %8 offset:1536\n\t"
          "s_waitcnt lgkmcnt(0)"
          : "=&v"(x0), "=&v"(x1), "=&v"(A0), "=&v"(B0), "=&v"(A1), "=&v"(B1)
          : "v"(xa), "v"(aa), "v"(ba));
      __builtin_amdgcn_sched_barrier(0);
      const v4i B0w = __builtin_shufflevector(B0, B0, 0, 1, -1, -1), B1w = __builtin_shufflevector(B1, B1, 0, 1, -1, -1);
      const v8i Aop[CB] = {__builtin_shufflevector(A0, B0w, 0, 1, 2, 3, 4, 5, -1, -1),
                           __builtin_shufflevector(A1, B1w, 0, 1, 2, 3, 4, 5, -1, -1)};
      const v4i X[2] = {x0, x1};
#pragma unroll
      for (int pb = 0; pb < PB; ++pb) {
        const v8i Bop = fp6_operand((uint32_t)X[pb][0], (uint32_t)X[pb][1], (uint32_t)X[pb][2]);
#pragma unroll
        for (int cb = 0; cb < CB; ++cb)
          acc[cb][pb] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(Aop[cb], Bop, first ? v16f{} : acc[cb][pb], 2,
                                                                        2, 0, 0, 0, 0);
      }
      return;
    }
    uint2 xw[PB];
    v4i A0, A1;
    if constexpr (PB == 4) {
      asm volatile(
          "ds_read_b64 %0, %6\n\t"
          "ds_read_b64 %1, %6 offset:512\n\t"
          "ds_read_b64 %2, %6 offset:1024\n\t"
          "ds_read_b64 %3, %6 offset:1536\n\t"
          "ds_read_b128 %4, %7\n\t"
          "ds_read_b128 %5, %7 offset:1024\n\t"
          "s_waitcnt lgkmcnt(0)"
          : "=&v"(xw[0]), "=&v"(xw[1]), "=&v"(xw[2]), "=&v"(xw[3]), "=&v"(A0), "=&v"(A1)
          : "v"(xa), "v"(aa));
    } else {
      asm volatile(
          "ds_read_b64 %0, %4\n\t"
          "ds_read_b64 %1, %4 offset:512\n\t"
          "ds_read_b128 %2, %5\n\t"
          "ds_read_b128 %3, %5 offset:1024\n\t"
          "s_waitcnt lgkmcnt(0)"
          : "=&v"(xw[0]), "=&v"(xw[1]), "=&v"(A0), "=&v"(A1)
          : "v"(xa), "v"(aa));
    }
    __builtin_amdgcn_sched_barrier(0);
    // E2M1 operands use the low four registers of each v8i (the rest is
    // ignored for this format)
    const v8i Aop[CB] = {__builtin_shufflevector(A0, A0, 0, 1, 2, 3, -1, -1, -1, -1),
                         __builtin_shufflevector(A1, A1, 0, 1, 2, 3, -1, -1, -1, -1)};
#pragma unroll
    for (int pb = 0; pb < PB; ++pb) {
      const uint32_t m = 0x33333333u;
      const v4i b = {(int)(xw[pb].x & m), (int)((xw[pb].x >> 2) & m), (int)(xw[pb].y & m), (int)((xw[pb].y >> 2) & m)};
      const v8i Bop = __builtin_shufflevector(b, b, 0, 1, 2, 3, -1, -1, -1, -1);
#pragma unroll
      for (int cb = 0; cb < CB; ++cb)
        acc[cb][pb] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
            Aop[cb], Bop, first ? (F32 ? c0[cb] : v16f{}) : acc[cb][pb], 4, 4, 0, 0, 0, 0);
    }
  };

  static_assert(S == 4, "the waits below count at most two younger fetches");
  // wait until K-block kb's loads have landed, y of this wave's fetches
  // (LPK loads or more each) being younger
  auto wait_younger = [&](int y) __attribute__((always_inline)) {
    if (y >= 2) __builtin_amdgcn_s_waitcnt(waitcnt_vm(2 * C::LPK));
    else if (y == 1) __builtin_amdgcn_s_waitcnt(waitcnt_vm(C::LPK));
    else __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
  };
  __syncthreads();  // the tile's constants are in LDS
  const int NS = KB / KS;  // ring stages (the host takes KS = 2 only for an even KB)
#pragma unroll
  for (int st = 0; st < S - 1; ++st)
    if (st < NS) fetch(st);
  if constexpr (F32) {
    // element r of block cb is channel 32 cb + 8 (r / 4) + 4 half + r % 4
    // of the wave's channels
#pragma unroll
    for (int cb = 0; cb < CB; ++cb)
#pragma unroll
      for (int qi = 0; qi < 4; ++qi) {
        const v4f b = *(const v4f *)(b4_area + wn * CB * 32 + cb * 32 + 8 * qi + 4 * half);
#pragma unroll
        for (int e = 0; e < 4; ++e) c0[cb][4 * qi + e] = kh == 0 ? b[e] : 0.0f;  // the bias once
      }
  }
  // stage 0 (NS >= 1)
  const bool steady0 = NS > S - 1;
  wait_younger(steady0 ? S - 2 : NS - 1);
  ring_barrier();
  if (steady0) fetch(S - 1);
  kblock(0, true);
  // steady state: K-block kb's loads were issued S - 1 fetches ago; at most
  // (S - 2) LPK of this wave's loads are younger
  int kb = 1;
  for (; kb + S - 1 < NS; ++kb) {
    __builtin_amdgcn_s_waitcnt(waitcnt_vm((S - 2) * C::LPK));
    ring_barrier();
    fetch((kb + S - 1) % S);
    kblock(kb % S, false);
  }
  // the last S - 1 K-blocks: no more fetches, the waits tighten
#pragma unroll
  for (int i = 0; i < S - 1; ++i) {
    if (kb >= NS) break;  // uniform
    wait_younger(NS - 1 - kb);
    ring_barrier();
    kblock(kb % S, false);
    ++kb;
  }

  if constexpr (KS == 2) {
    // group 1's accumulators into group 0's: chunk c (4 values) of wave w at
    // ((w 16 + c) 64 + lane) 16 bytes, over the ring, which every wave has
    // finished reading at the first barrier
    __syncthreads();
    float *red = (float *)lds;
    if (kh == 1) {
#pragma unroll
      for (int cb = 0; cb < CB; ++cb)
#pragma unroll
        for (int pb = 0; pb < PB; ++pb)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int c = (cb * PB + pb) * 4 + q;
            *(v4f *)(red + ((wave * 16 + c) * 64 + lane) * 4) =
                v4f{acc[cb][pb][4 * q], acc[cb][pb][4 * q + 1], acc[cb][pb][4 * q + 2], acc[cb][pb][4 * q + 3]};
          }
    }
    __syncthreads();
    if (kh == 1) return;
#pragma unroll
    for (int cb = 0; cb < CB; ++cb)
#pragma unroll
      for (int pb = 0; pb < PB; ++pb)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int c = (cb * PB + pb) * 4 + q;
          const v4f r = *(const v4f *)(red + ((wave * 16 + c) * 64 + lane) * 4);
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[cb][pb][4 * q + e] += r[e];  // exact (multiples of 1/4 below 2^22)
        }
  }

  // ---- epilogue
  const int64_t mbase = (int64_t)pt * TM + wm * PB * 32;
  if constexpr (DUMP) {
    const int64_t outC = (int64_t)G * a.cout;
#pragma unroll
    for (int cb = 0; cb < CB; ++cb)
#pragma unroll
      for (int pb = 0; pb < PB; ++pb) {
        const int64_t mp = mbase + pb * 32 + l32;
        if (mp >= geo.M) continue;
        int32_t *dst = a.acc_dump + mp * outC + (int64_t)gd * a.cout + cbk * TN + wn * CB * 32 + cb * 32 + 4 * half;
#pragma unroll
        for (int qi = 0; qi < 4; ++qi) {
          v4i dv;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            // exact: |t| < 2^23 (F32: the accumulator is (t + bias) / 4, each term below 2^22)
            const float b = F32 ? b4_area[wn * CB * 32 + cb * 32 + 8 * qi + 4 * half + e] : 0.0f;
            dv[e] = (int)((acc[cb][pb][4 * qi + e] - b) * (B == 2 ? 4.0f : 8.0f));
          }
          *(v4i *)(dst + 8 * qi) = dv;
        }
      }
  }
  // this lane's shortcut codes: pixel block pb, channel block cb at
  // ra + pb 32 RPX + 8 cb (read per channel block by the epilogue)
  const uint32_t ra = RB == 2 ? lds_base + RING + (uint32_t)((wm * PB * 32 + l32) * C::RPX + wn * CB * 8) : 0u;
  uint32_t rw[CB][PB][2] = {};
  epilogue_fast_bo<B, CB, PB, RB, v16f, true, F32>(a, geo, acc, rw, mbase, g, gd, cbk * TN + wn * CB * 32, l32, half,
                                                     rq_area + wn * CB * 32, rm_area + (RB ? wn * CB * 32 : 0), ra,
                                                     32 * C::RPX, sc_area + wn * CB * 32);
}

template <int CB, int PB, int WN, int WM, int RB, bool DUMP, int S, bool F32, int KS = 1>
__global__ __launch_bounds__(WN * WM * 64 * KS, 2) void conv_fp4_kernel(ConvArgs a, Geo geo, int npt, int ncb, int nch) {
  conv_fpx_tile<CB, PB, WN, WM, RB, DUMP, S, 2, F32, KS>(a, geo, npt, ncb, nch);
}
template <int CB, int PB, int WN, int WM, bool DUMP, int S>
__global__ __launch_bounds__(WN * WM * 64, 2) void conv_fp6_kernel(ConvArgs a, Geo geo, int npt, int ncb, int nch) {
  conv_fpx_tile<CB, PB, WN, WM, 0, DUMP, S, 3>(a, geo, npt, ncb, nch);
}

// ---------------------------------------------------------------- Eq. 4 bit decomposition
// The M-bit baseline of Section 3.2 run on the 2-bit (FP4) matrix cores:
// every unsigned M-bit activation code x and signed M-bit weight w (M = 4,
// 6, 8) is split into G = M / 2 2-bit chunks, x = sum_i 4^i x_i and
// w = sum_j 4^j w_j (w_j unsigned for j < G - 1, the top chunk signed), and
// each MAC becomes the G^2 chunk products of Eq. 4, 4^(i+j) x_i w_j, summed
// exactly.  A K-block (tap, 64 input channels) stages the pixels' M-bit
// codes (32 or 64 bytes a pixel) and the G chunk slabs of the weights
// (prepack_bd_kernel); a lane then builds its G activation chunk operands in
// registers and runs G^2 FP4 MFMAs per 32 x 32 block, the factor 4^(i+j)
// given as the E8M0 scale of the activation operand.  Operands are E2M1 of
// c / 2 (chunks 0..3 and the top chunk -2..1), so the fp32 accumulator
// holds T / 4 with T the integer sum; M = 8 keeps the pairs with i + j >= 3
// in a second accumulator scaled by 4^-3, so that each stays below 2^24 in T
// (bd_applies checks the bounds).  Tiles as conv_fpx_tile (128 x 128,
// XCD-contiguous runs in the chunked order).  Epilogue in fp64: lo + 64 hi,
// plus the identity shortcut rm c / 4 (M-bit codes), then the FP4-scaled
// requant constants.  A fused projection adds its own decomposed K-blocks.
namespace bd {
template <int M, int WN>
struct Cfg {
  static constexpr int GC = M / 2;  // chunks of a code
  static constexpr int CB = 2, PB = 2, WM = 2;  // WN = 1: 64-channel tiles, 2: 128
  static constexpr int NT = WN * WM * 64;
  static constexpr int TN = WN * CB * 32, TM = WM * PB * 32;
  static constexpr int XB = M == 4 ? 32 : 64;  // bytes of a pixel's 64-code K-block
  static constexpr int Q = XB / 32;            // 16-byte pieces of a lane half
  static constexpr int WST = TN / 32 * GC * kSlab4;
  static constexpr int XST = TM * XB;
  static constexpr int SST = WST + XST;
  static constexpr int WP = WST / 16, XP = XST / 16;
  static_assert(WP % NT == 0 && XP % NT == 0, "every thread loads whole pieces");
  static constexpr int WL = WP / NT, XL = XP / NT;
  static constexpr int LPK = WL + XL;  // loads per K-block, the same for every wave
  static constexpr bool SPLIT = M == 8;
  static constexpr int S = 3;  // ring stages
};
// Code index (within a lane's 32) of operand nibble n: M = 4 codes are
// nibbles already; byte codes pair dwords 2r and 2r + 1 into one nibble word.
__host__ __device__ inline int bd_code(int M, int n) {
  return M == 4 ? n : 8 * (n >> 3) + 4 * (n & 1) + ((n >> 1) & 3);
}
}  // namespace bd

// Weights -> [G][cout/32][kb_total][GC chunk slabs of 1 KB][half][ch][16 B]:
// nibble n of lane (ch, half) of slab j holds E2M1 of w_j / 2 for the
// K-block code 32 half + bd_code(M, n).  One thread per 16-byte lane operand.
__global__ void prepack_bd_kernel(ConvArgs a, Geo geo, uint8_t *wp) {
  const int M = a.w_bits, GC = M / 2, sb = M == 4 ? 4 : 8;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int nc32 = a.cout / 32;
  const int64_t total = (int64_t)a.in.groups * nc32 * geo.kb_total * GC * 64;
  if (t >= total) return;
  const int lane = (int)(t & 63), j = (int)((t >> 6) % GC);
  const int64_t rest = (t >> 6) / GC;
  const int kb = (int)(rest % geo.kb_total);
  const int64_t r2 = rest / geo.kb_total;
  const int cblk = (int)(r2 % nc32), g = (int)(r2 / nc32);
  const int half = lane >> 5, k = cblk * 32 + (lane & 31);
  const int gd = (g + a.shuffle) % a.in.groups;
  const int kbytes = 64 * sb / 8;  // bytes of a K-block of one channel
  const uint8_t *p = kb < geo.kb_main ? a.w + ((int64_t)g * a.cout + k) * geo.w_ch + (int64_t)kb * kbytes
                                      : a.proj_w + ((int64_t)gd * a.cout + k) * geo.pw_ch +
                                            (int64_t)(kb - geo.kb_main) * kbytes;
  uint32_t o[4] = {0, 0, 0, 0};
  for (int n = 0; n < 32; ++n) {
    const int m = 32 * half + bd::bd_code(M, n);
    const int raw = sb == 4 ? (p[m >> 1] >> (4 * (m & 1))) & 15 : p[m];
    const int w = (raw << (32 - M)) >> (32 - M);  // sign-extend the M-bit code
    int c = w >> (2 * j);                          // chunk j: top chunk signed, others 0..3
    if (j < GC - 1) c &= 3;
    const uint32_t e = j < GC - 1 ? (uint32_t)c                        // E2M1 of c / 2 for c = 0..3
                                  : (0x9A10u >> (4 * (c & 3))) & 15u;  // -2, -1, 0, 1 -> -1, -0.5, 0, 0.5
    o[n >> 3] |= e << (4 * (n & 7));
  }
  *(uint4 *)(wp + t * 16) = make_uint4(o[0], o[1], o[2], o[3]);
}

// Chunk i of a lane's 32 M-bit codes (raw: 4 words of nibbles, or 8 words of
// bytes) as an E2M1 operand of c_i / 2 in bd_code order.
template <int M>
__device__ inline v8i bd_operand(const uint32_t (&raw)[M == 4 ? 4 : 8], int i) {
  v8i d;
  if constexpr (M == 4) {
#pragma unroll
    for (int q = 0; q < 4; ++q) d[q] = (int)((raw[q] >> (2 * i)) & 0x33333333u);
  } else {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const uint32_t e = (raw[2 * r] >> (2 * i)) & 0x03030303u, o = (raw[2 * r + 1] >> (2 * i)) & 0x03030303u;
      d[r] = (int)(e | (o << 4));
    }
  }
  d[4] = d[5] = d[6] = d[7] = 0;
  return d;
}

template <int M, int WN, int RB, bool DUMP>
__global__ __launch_bounds__(WN * 128, 2) void conv_bitdecomp_kernel(ConvArgs a, Geo geo, int npt, int ncb, int nch) {
  using C = bd::Cfg<M, WN>;
  constexpr int NT = C::NT, TN = C::TN, TM = C::TM, WST = C::WST, SST = C::SST, S = C::S, GC = C::GC;
  // (local copies: a member of the dependent C inside a builtin's argument
  // costs the host pass this kernel's launch stub)
  constexpr int CB = C::CB, PB = C::PB, Q = C::Q, XB = C::XB;
  constexpr int BO = M == 4 ? 4 : 8;  // output storage bits (6-bit codes as bytes)
  extern __shared__ __attribute__((aligned(1024))) uint8_t lds[];
  RqConst *rq_area = (RqConst *)(lds + S * SST);
  int32_t *rm_area = (int32_t *)(rq_area + TN);

  if (int64_flag(a, geo)) return;  // the general partner takes the layer
  const int G = a.in.groups;
  const int T = npt * ncb * G;
  const int x8 = (int)(blockIdx.x & 7), jx = (int)(blockIdx.x >> 3);
  const int Tq = T >> 3, Tr = T & 7;
  if (jx >= Tq + (x8 < Tr ? 1 : 0)) return;  // no barrier yet
  const int t = x8 * Tq + min(x8, Tr) + jx;
  const TileIt it = tile_at(t, npt, ncb * G, nch);
  const int pt = it.pt, cbk = it.combo % ncb, g = it.combo / ncb;
  const int gd = (g + a.shuffle) % G;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = uniform_int(tid >> 6);
  const int l32 = lane & 31, half = lane >> 5;
  const int wn = wave / C::WM, wm = wave % C::WM;
  const int KB = geo.kb_total, KM = geo.kb_main;

  const int64_t ch0 = (int64_t)g * a.cout + cbk * TN;
  for (int c = tid; c < TN; c += NT) {
    rq_area[c] = geo.rq[ch0 + c];
    rm_area[c] = RB != 0 ? a.res_mult[ch0 + c] : 0;
  }
  typedef __attribute__((address_space(3))) void *lds_ptr;
  const uint32_t lds_base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t *)lds;
  const auto rw_src = make_rsrc(geo.wp, (int64_t)G * a.cout * KB * GC * (kSlab4 / 32));
  const auto rin = make_rsrc(a.in.data, a.in.bytes);
  const auto rpj = a.proj.data ? make_rsrc(a.proj.data, a.proj.bytes)
                               : make_rsrc(a.in.data, 0);
  const int pixb = (int)a.in.pixel, rowb = a.in.w * pixb;

  // ---- fetch pieces.  Weights: piece c = tid + i NT of the tile's K-block:
  // 32-channel block c / (64 GC), chunk slab (c / 64) % GC, lane c % 64.
  // Activations: piece q = tid + i NT: 32-pixel block (q / 64) / Q, part
  // (q / 64) % Q (16 bytes) of lane half (q / 32) & 1, pixel q % 32.
  uint32_t woff[C::WL];
#pragma unroll
  for (int i = 0; i < C::WL; ++i) {
    const int c = tid + i * NT;
    woff[i] = (uint32_t)((((int64_t)g * (a.cout / 32) + cbk * (TN / 32) + c / (64 * GC)) * KB) * GC * kSlab4 +
                         (c % (64 * GC)) * 16);
  }
  const int HW = a.ho * a.wo;
  const float inv_hw = geo.inv_hw, inv_wo = geo.inv_wo;
  int off0[C::XL], poff[C::XL];
  uint32_t tmask[C::XL];
#pragma unroll
  for (int i = 0; i < C::XL; ++i) {
    const int q = tid + i * NT, bp = q >> 6;
    const int part = bp % Q, m = pt * TM + 32 * (bp / Q) + (q & 31);
    const int hoff = XB / 2 * ((q >> 5) & 1) + 16 * part;  // bytes of the lane half's part
    const bool valid = m < geo.M;
    const int mm = valid ? m : 0;
    const int n = fdiv(mm, HW, inv_hw);
    const int rem = mm - n * HW;
    const int oy = fdiv(rem, a.wo, inv_wo);
    const int ox = rem - oy * a.wo;
    const int iy0 = oy * a.stride - a.pad, ix0 = ox * a.stride - a.pad;
    off0[i] = ((n * a.in.h + iy0) * a.in.w + ix0) * pixb + g * (int)a.in.gstride + hoff;
    const int xlo = max(0, -ix0), xhi = min(a.kw, a.in.w - ix0);
    const uint32_t below = xhi >= 32 ? 0xffffffffu : ((1u << max(xhi, 0)) - 1u);
    const uint32_t cols = xhi > xlo ? (below & ~((1u << xlo) - 1u)) : 0u;
    const int ylo = max(0, -iy0), yhi = min(a.kh, a.in.h - iy0);
    uint32_t mk = 0;
    for (int ky = ylo; ky < yhi; ++ky) mk |= cols << (ky * a.kw);
    tmask[i] = valid ? mk : 0u;
    poff[i] = (a.proj.data && valid)
                  ? (((n * a.proj.h + oy * a.proj_stride) * a.proj.w + ox * a.proj_stride) * (int)a.proj.pixel +
                     gd * (int)a.proj.gstride + hoff)
                  : (int)kOob;
  }
  int f_kb = 0, f_c = 0, f_tap = 0, f_kx = 0, f_tapoff = 0;
  uint32_t vo[C::XL];
  auto tap_offsets = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < C::XL; ++i) vo[i] = ((tmask[i] >> f_tap) & 1u) ? (uint32_t)(off0[i] + f_tapoff) : kOob;
  };
  tap_offsets();
  auto fetch = [&](int st) __attribute__((always_inline)) {
    uint8_t *ws = lds + st * SST;
#pragma unroll
    for (int i = 0; i < C::WL; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rw_src, (lds_ptr)(ws + i * NT * 16 + wave * 1024), 16, (int)woff[i],
                                               f_kb * GC * kSlab4, 0, 0);
    if (f_kb < KM) {
#pragma unroll
      for (int i = 0; i < C::XL; ++i)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rin, (lds_ptr)(ws + WST + i * NT * 16 + wave * 1024), 16, (int)vo[i],
                                                 f_c * XB, 0, 0);
    } else {
#pragma unroll
      for (int i = 0; i < C::XL; ++i)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rpj, (lds_ptr)(ws + WST + i * NT * 16 + wave * 1024), 16,
                                                 (int)poff[i], (f_kb - KM) * XB, 0, 0);
    }
    ++f_kb;
    if (++f_c == geo.cpb) {  // next tap
      f_c = 0;
      ++f_tap;
      f_tapoff += pixb;
      if (++f_kx == a.kw) {
        f_kx = 0;
        f_tapoff += rowb - a.kw * pixb;
      }
      tap_offsets();
    }
  };

  // ---- compute side
  v16f acc[CB][PB], ach[C::SPLIT ? CB : 1][C::SPLIT ? PB : 1];
#pragma unroll
  for (int cb = 0; cb < CB; ++cb)
#pragma unroll
    for (int pb = 0; pb < PB; ++pb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        acc[cb][pb][r] = 0.f;
        if constexpr (C::SPLIT) ach[cb][pb][r] = 0.f;
      }
  // this lane's operands in stage 0: weight slab j of channel block cb at
  // ((wn CB + cb) GC + j) KB; activation part p of pixel block pb at
  // ((wm PB + pb) Q + p) KB
  const uint32_t aaddr0 = lds_base + (uint32_t)(wn * CB * GC * kSlab4 + lane * 16);
  const uint32_t xaddr0 = lds_base + WST + (uint32_t)(wm * PB * Q * 1024 + lane * 16);
  auto kblock = [&](int st) __attribute__((always_inline)) {
    const uint32_t aa = aaddr0 + st * SST, xa = xaddr0 + st * SST;
    // operand reads as asm (the compiler would wait for every staging load
    // before an LDS read it sees), one wait, then each value is tied to it
    v4i A[CB][GC], X[PB][Q];
#pragma unroll
    for (int cb = 0; cb < CB; ++cb)
#pragma unroll
      for (int j = 0; j < GC; ++j)
        asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(A[cb][j]) : "v"(aa), "i"((cb * GC + j) * kSlab4));
#pragma unroll
    for (int pb = 0; pb < PB; ++pb)
#pragma unroll
      for (int p = 0; p < Q; ++p)
        asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(X[pb][p]) : "v"(xa), "i"((pb * Q + p) * 1024));
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
    for (int cb = 0; cb < CB; ++cb)
#pragma unroll
      for (int j = 0; j < GC; ++j) asm volatile("" : "+v"(A[cb][j]));
    uint32_t raw[PB][M == 4 ? 4 : 8];
#pragma unroll
    for (int pb = 0; pb < PB; ++pb)
#pragma unroll
      for (int p = 0; p < Q; ++p) {
        asm volatile("" : "+v"(X[pb][p]));
#pragma unroll
        for (int e = 0; e < 4; ++e) raw[pb][4 * p + e] = (uint32_t)X[pb][p][e];
      }
#pragma unroll
    for (int i = 0; i < GC; ++i)
#pragma unroll
      for (int pb = 0; pb < PB; ++pb) {
        const v8i Bop = bd_operand<M>(raw[pb], i);
#pragma unroll
        for (int j = 0; j < GC; ++j)
#pragma unroll
          for (int cb = 0; cb < CB; ++cb) {
            const v8i Aop = __builtin_shufflevector(A[cb][j], A[cb][j], 0, 1, 2, 3, -1, -1, -1, -1);
            const bool hi = C::SPLIT && i + j >= 3;
            const int sc = 127 + 2 * (i + j) - (hi ? 6 : 0);  // E8M0 of 4^(i+j) (4^(i+j-3) for the second sum)
            if (hi)
              ach[cb][pb] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(Aop, Bop, ach[cb][pb], 4, 4, 0, 127, 0, sc);
            else
              acc[cb][pb] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(Aop, Bop, acc[cb][pb], 4, 4, 0, 127, 0, sc);
          }
      }
  };

  __syncthreads();  // the tile's constants are in LDS
#pragma unroll
  for (int st = 0; st < S - 1; ++st)
    if (st < KB) fetch(st);
  int kb = 0;
  for (; kb + S - 1 < KB; ++kb) {
    __builtin_amdgcn_s_waitcnt(waitcnt_vm((S - 2) * C::LPK));
    ring_barrier();
    fetch((kb + S - 1) % S);
    kblock(kb % S);
  }
#pragma unroll
  for (int i = 0; i < S - 1; ++i) {
    if (kb >= KB) break;  // uniform
    if (KB - 1 - kb >= 1) __builtin_amdgcn_s_waitcnt(waitcnt_vm(C::LPK));
    else __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
    ring_barrier();
    kblock(kb % S);
    ++kb;
  }

  // ---- epilogue (fp64): v = T / 4 (+ the shortcut rm c / 4), then
  // q = min(trunc(v s + o), 2^out_bits - 1) with the FP4 requant constants
  const int64_t mbase = (int64_t)pt * TM + wm * PB * 32;
  const int64_t outC = (int64_t)G * a.cout;
  const uint32_t qmax = (1u << a.out.bits) - 1u;
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    const int kc = cbk * TN + wn * CB * 32 + cb * 32;  // first channel of this 32-channel block
    const int lc = wn * CB * 32 + cb * 32;             // the same within the tile
    uint32_t qv[PB][4];
#pragma unroll
    for (int pb = 0; pb < PB; ++pb) {
      const int64_t mp = mbase + pb * 32 + l32;
      const bool live = mp < geo.M;
#pragma unroll
      for (int qi = 0; qi < 4; ++qi) {
        const int cq = 8 * qi + 4 * half;
        int rc[4] = {0, 0, 0, 0};
        if constexpr (RB < 0)
          row_quad(a.res.data + (live ? mp : 0) * a.res.pixel + (int64_t)gd * a.res.gstride, kc + cq, a.res.bits, rc);
        uint32_t qword = 0;
        v4i dv;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          double v = (double)acc[cb][pb][4 * qi + e];
          if constexpr (C::SPLIT) v += 64.0 * (double)ach[cb][pb][4 * qi + e];
          dv[e] = (int)(4.0 * v);  // T: exact, |T| < 2^31
          if constexpr (RB < 0) v += 0.25 * (double)rm_area[lc + cq + e] * (double)rc[e];
          const RqConst k = rq_area[lc + cq + e];
          const double d = __builtin_fma(v, k.s, k.o);
          uint32_t q;
          asm("v_cvt_u32_f64 %0, %1" : "=v"(q) : "v"(d));
          qword |= min(q, qmax) << (BO * e);
        }
        qv[pb][qi] = qword;
        if constexpr (DUMP)
          if (live) *(v4i *)(a.acc_dump + mp * outC + (int64_t)gd * a.cout + kc + cq) = dv;
      }
    }
#pragma unroll
    for (int pb = 0; pb < PB; ++pb) {
      const int64_t mp = mbase + pb * 32 + l32;
      // as in epilogue_fast_bo: after the swaps every lane holds its 32
      // channels' quads in order (16 of them per lane half)
      const auto p0 = __builtin_amdgcn_permlane32_swap(qv[pb][0], qv[pb][2], false, false);
      const auto p1 = __builtin_amdgcn_permlane32_swap(qv[pb][1], qv[pb][3], false, false);
      const uint32_t Qw[4] = {p0[0], p0[1], p1[0], p1[1]};
      if (mp >= geo.M) continue;
      uint32_t *cw = (uint32_t *)(a.out.data + mp * a.out.pixel + (int64_t)gd * a.out.gstride) + (int64_t)(kc >> 5) * BO +
                     half * (BO / 2);
      if constexpr (BO == 4) *(uint2 *)cw = make_uint2(Qw[0] | (Qw[1] << 16), Qw[2] | (Qw[3] << 16));
      else *(uint4 *)cw = make_uint4(Qw[0], Qw[1], Qw[2], Qw[3]);
    }
  }
}

// ---------------------------------------------------------------- launch
bool is_stem(const ConvArgs &a) {
  return a.in.bits == 8 && a.in.is_signed && a.w_bits == 8 && a.in.row == 4 && a.kw <= 8 &&
         !a.proj.data;
}

Geo make_geo(const ConvArgs &a) {
  Geo geo{};
  geo.M = a.out.n * a.ho * a.wo;
  geo.inv_hw = a.ho * a.wo > 0 ? 1.0f / (float)(a.ho * a.wo) : 0.0f;
  geo.inv_wo = a.wo > 0 ? 1.0f / (float)a.wo : 0.0f;
  if (is_stem(a)) {
    geo.kb_main = (a.kh + 1) / 2;  // two filter rows per K-block
    geo.kb_total = geo.kb_main;
    geo.scale = 1;
  } else {
    geo.cpb = a.in.cpg / 64;
    geo.kb_main = a.kh * a.kw * geo.cpb;
    geo.kb_total = geo.kb_main + (a.proj.data ? a.proj.cpg / 64 : 0);
    geo.w_ch = (int64_t)a.kh * a.kw * row_bytes(a.in.cpg, a.w_bits);
    geo.pw_ch = a.proj.data ? row_bytes(a.proj.cpg, a.w_bits) : 0;
    geo.scale = a.in.bits == 2 ? 16 : 1;
  }
  return geo;
}

size_t lds_bytes(const Geo &geo, int cb) { return (size_t)geo.kb_total * cb * kSlab + (size_t)cb * 32 * sizeof(RqConst); }

// Largest channel block (32 or 64 channels) whose filter fits LDS, 0 if
// none.  Two blocks per wave share every activation load and unpack.
int pick_cb(const ConvArgs &a, const Geo &geo) {
  if (a.cout % 64 == 0 && lds_bytes(geo, 2) <= kLdsBudget) return 2;
  if (lds_bytes(geo, 1) <= kLdsBudget) return 1;
  return 0;
}

template <typename K>
hipError_t launch_persistent(K kern, const ConvArgs &a, const Geo &geo, int cb, int pb, hipStream_t s) {
  const size_t lds = lds_bytes(geo, cb);
  hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, kLdsBudget);
  if (e != hipSuccess) return e;
  const int tiles = (int)((geo.M + pb * 32 - 1) / (pb * 32));
  const int combos = (a.cout / (cb * 32)) * a.in.groups;
  const int per_cu = (int)std::min<size_t>(2, kLdsBudget / std::max<size_t>(lds, 1));
  int gx = std::max(1, (256 * per_cu + combos - 1) / combos);
  gx = std::min(gx, (tiles + kNW - 1) / kNW);
  dim3 grid((unsigned)gx, (unsigned)(a.cout / (cb * 32)), (unsigned)a.in.groups);
  hipLaunchKernelGGL(kern, grid, dim3(kNW * 64), lds, s, a, geo, tiles);
  return hipGetLastError();
}

// Starts the fast build, the general build or both (epi -1: which one
// applies is only known on the device; the other returns at once).
template <typename KF, typename KG>
hipError_t launch_pair(KF kfast, KG kgen, int epi, const ConvArgs &a, const Geo &geo, int cb, int pb,
                       hipStream_t s) {
  hipError_t e = hipSuccess;
  if (epi != 1) e = launch_persistent(kfast, a, geo, cb, pb, s);
  if (e == hipSuccess && epi != 0) e = launch_persistent(kgen, a, geo, cb, pb, s);
  return e;
}

template <int B, int CB, int PB>
hipError_t launch_grouped(const ConvArgs &a, const Geo &geo, int epi, hipStream_t s) {
  if (!a.res.data)
    return launch_pair(conv_grouped_kernel<B, CB, PB, 0, false>, conv_grouped_kernel<B, CB, PB, 0, true>, epi, a,
                       geo, CB, PB, s);
  if (a.res.bits == 2)
    return launch_pair(conv_grouped_kernel<B, CB, PB, 2, false>, conv_grouped_kernel<B, CB, PB, 2, true>, epi, a,
                       geo, CB, PB, s);
  return launch_persistent(conv_grouped_kernel<B, CB, PB, -1, true>, a, geo, CB, PB, s);
}

template <int CB, int PB>
hipError_t launch_stem(const ConvArgs &a, const Geo &geo, int epi, hipStream_t s) {
  if (!a.res.data)
    return launch_pair(conv_stem_kernel<CB, PB, 0, false>, conv_stem_kernel<CB, PB, 0, true>, epi, a, geo, CB, PB,
                       s);
  return launch_persistent(conv_stem_kernel<CB, PB, -1, true>, a, geo, CB, PB, s);
}

template <int B>
hipError_t dispatch_bits(const ConvArgs &a, const Geo &geo, int cb, int pb, int epi, hipStream_t s) {
  (void)pb;  // one 32-pixel block per wave
  // 8-bit codes with a shortcut: the 64-channel general build would spill
  if constexpr (B == 8)
    if (a.res.data) return launch_grouped<B, 1, 1>(a, geo, epi, s);
  return cb == 2 ? launch_grouped<B, 2, 1>(a, geo, epi, s) : launch_grouped<B, 1, 1>(a, geo, epi, s);
}

// Largest magnitude of a code of the given width and sign.
int64_t code_max(int bits, int is_signed) {
  return is_signed ? ((int64_t)1 << (bits - 1)) : (((int64_t)1 << bits) - 1);
}

// Bound on |accumulator|: every product of the main and projection
// contractions at its largest.
int64_t acc_bound_of(const ConvArgs &a) {
  int64_t b = (int64_t)a.kh * a.kw * a.in.cpg * code_max(a.in.bits, a.in.is_signed) * code_max(a.w_bits, 1);
  if (a.proj.data) b += (int64_t)a.proj.cpg * code_max(a.proj.bits, 0) * code_max(a.w_bits, 1);
  return b;
}

}  // namespace

bool fp4_applies(const ConvArgs &a);
bool fp6_applies(const ConvArgs &a);
bool bd_applies(const ConvArgs &a);
size_t bd_offset(const ConvArgs &a);
bool tile_kernel_applies(const ConvArgs &a);
bool stem_tile_applies(const ConvArgs &a);
bool stem_rows(const ConvArgs &a);
size_t stem_rows_offset(const ConvArgs &a);

bool conv_mfma_general_fits(const ConvArgs &a) { return pick_cb(a, make_geo(a)) > 0; }

bool conv_mfma_supported(const ConvArgs &a) {
  if (a.cout % 32 != 0) return false;
  const int64_t lim = (int64_t)1 << 30;
  auto bytes = [](const ActView &v) { return v.data ? v.bytes : 0; };
  if (bytes(a.in) >= lim || bytes(a.out) >= lim || bytes(a.res) >= lim || bytes(a.proj) >= lim) return false;
  if ((int64_t)a.out.n * a.ho * a.wo >= (1 << 24)) return false;
  if (!is_stem(a)) {
    const int b = a.in.bits;
    if (a.in.is_signed || (b != 2 && b != 3 && b != 4 && b != 6 && b != 8) || a.w_bits != b) return false;
    if (a.in.cpg % 64 != 0 || a.kh * a.kw > 32) return false;
    if (a.proj.data && (a.proj.bits != b || a.proj.cpg % 64 != 0 || a.proj.is_signed)) return false;
  }
  // the general build needs the filter in LDS; layers longer than that
  // still run on the tiled kernel (its fast epilogue)
  return pick_cb(a, make_geo(a)) > 0 || tile_kernel_applies(a) || stem_tile_applies(a);
}

ConvPlan conv_mfma_plan(const ConvArgs &a) {
  ConvPlan p{};
  const Geo geo = make_geo(a);
  p.w_bytes = (size_t)a.in.groups * a.cout * geo.kb_total * 64;
  if (!is_stem(a) && a.in.bits >= 6) p.w_bytes += (size_t)a.in.groups * a.cout * 4;  // Geo::acc0
  p.thr_bytes = (size_t)a.in.groups * a.cout * sizeof(RqConst) + 16;  // + int64-path flag
  if (stem_rows(a)) p.w_bytes += (size_t)a.cout * sp::KH * 32;  // the filter-row copy
  if (fp6_applies(a)) {  // FP6 slabs and constants after the int8 ones
    p.w_bytes += (size_t)a.in.groups * a.cout * geo.kb_total * 48;
    p.thr_bytes *= 2;
  }
  if (bd_applies(a)) {  // the decomposition's chunk slabs and FP4-scaled constants
    p.w_bytes = bd_offset(a) + (size_t)a.in.groups * a.cout * geo.kb_total * (a.in.bits / 2) * 32;
    p.thr_bytes *= 2;
  }
  if (fp4_applies(a)) {  // FP4 slabs and constants after the int8 ones (the general build keeps those)
    p.w_bytes += (size_t)a.in.groups * a.cout * geo.kb_total * 32;
    p.thr_bytes *= 2;
    p.thr_bytes += (size_t)a.in.groups * a.cout * 12 + 16;  // fp32 scale, bias / 4, res_mult / 4, flag
  }
  return p;
}

hipError_t launch_conv_prepare(const ConvArgs &a, uint8_t *wp, int32_t *thr, hipStream_t s) {
  const Geo geo = make_geo(a);
  const int64_t chunks = (int64_t)a.in.groups * (a.cout / 32) * geo.kb_total * 128;
  const unsigned grid = (unsigned)((chunks + 255) / 256);
  if (is_stem(a)) {
    hipLaunchKernelGGL((prepack_kernel<8, true>), dim3(grid), dim3(256), 0, s, a, geo, wp);
    if (stem_rows(a)) {
      const int64_t pieces = (int64_t)a.cout * sp::KH * 2;
      hipLaunchKernelGGL(prepack_stem_rows_kernel, dim3((unsigned)((pieces + 255) / 256)), dim3(256), 0, s, a,
                         wp + stem_rows_offset(a));
    }
  } else {
    switch (a.in.bits) {
      case 2: hipLaunchKernelGGL((prepack_kernel<2, false>), dim3(grid), dim3(256), 0, s, a, geo, wp); break;
      case 3: hipLaunchKernelGGL((prepack_kernel<3, false>), dim3(grid), dim3(256), 0, s, a, geo, wp); break;
      case 4: hipLaunchKernelGGL((prepack_kernel<4, false>), dim3(grid), dim3(256), 0, s, a, geo, wp); break;
      case 6: case 8:
        hipLaunchKernelGGL((prepack_kernel<8, false>), dim3(grid), dim3(256), 0, s, a, geo, wp);
        hipLaunchKernelGGL(wsum_kernel, dim3((unsigned)((a.in.groups * a.cout + 255) / 256)), dim3(256), 0, s, a,
                           geo, (int32_t *)(wp + (size_t)a.in.groups * a.cout * geo.kb_total * 64));
        break;
      default: return hipErrorNotSupported;
    }
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t acc_bound = acc_bound_of(a);
  const int res_max = a.res.data ? (int)code_max(a.res.bits, 0) : 0;
  const int nch = a.in.groups * a.cout;
  RqConst *rq = (RqConst *)thr;
  const int lscale = geo.scale == 16 ? 4 : 0;  // the int8 accumulator is 16 t for 2-bit codes
  hipLaunchKernelGGL(requant_prep_kernel, dim3(1), dim3(256), 0, s, a.mult, a.shift, a.bias, a.res.data ? a.res_mult : nullptr,
                     res_max, nch, lscale, acc_bound, rq, (int32_t *)(rq + nch));
  e = hipGetLastError();
  if (e == hipSuccess && bd_applies(a)) {
    const int64_t lanes = (int64_t)a.in.groups * (a.cout / 32) * geo.kb_total * (a.in.bits / 2) * 64;
    hipLaunchKernelGGL(prepack_bd_kernel, dim3((unsigned)((lanes + 255) / 256)), dim3(256), 0, s, a, geo,
                       wp + bd_offset(a));
    RqConst *rqb = rq + nch + 1;  // the decomposition's accumulator is T / 4
    hipLaunchKernelGGL(requant_prep_kernel, dim3(1), dim3(256), 0, s, a.mult, a.shift, a.bias,
                       a.res.data ? a.res_mult : nullptr, res_max, nch, -2, acc_bound, rqb, (int32_t *)(rqb + nch));
    return hipGetLastError();
  }
  if (e == hipSuccess && fp6_applies(a)) {
    const int64_t lanes = (int64_t)a.in.groups * (a.cout / 32) * geo.kb_total * 64;
    hipLaunchKernelGGL(prepack_fp6_kernel, dim3((unsigned)((lanes + 255) / 256)), dim3(256), 0, s, a, geo,
                       wp + (size_t)a.in.groups * a.cout * geo.kb_total * 64);
    RqConst *rq6 = rq + nch + 1;  // the FP6 accumulator is t / 8
    hipLaunchKernelGGL(requant_prep_kernel, dim3(1), dim3(256), 0, s, a.mult, a.shift, a.bias, nullptr, 0, nch, -3,
                       acc_bound, rq6, (int32_t *)(rq6 + nch));
    return hipGetLastError();
  }
  if (e != hipSuccess || !fp4_applies(a)) return e;
  const int64_t pieces = (int64_t)a.in.groups * (a.cout / 32) * geo.kb_total * 64;
  hipLaunchKernelGGL(prepack_fp4_kernel, dim3((unsigned)((pieces + 255) / 256)), dim3(256), 0, s, a, geo,
                     wp + (size_t)a.in.groups * a.cout * geo.kb_total * 64);
  RqConst *rq4 = rq + nch + 1;  // the FP4 accumulator is t / 4
  hipLaunchKernelGGL(requant_prep_kernel, dim3(1), dim3(256), 0, s, a.mult, a.shift, a.bias, a.res.data ? a.res_mult : nullptr,
                     res_max, nch, -2, acc_bound, rq4, (int32_t *)(rq4 + nch));
  float *f32c = (float *)(rq4 + nch + 1);
  hipLaunchKernelGGL(requant_prep_f32_kernel, dim3(1), dim3(256), 0, s, a.mult, a.shift, a.bias,
                     a.res.data ? a.res_mult : nullptr, res_max, nch, acc_bound, f32c, f32c + nch, f32c + 2 * nch,
                     (int32_t *)(f32c + 3 * nch));
  return hipGetLastError();
}

bool conv_mfma_pads_input(const ConvArgs &a) { return is_stem(a) && a.pad > 0; }

bool conv_mfma_f32(const ConvArgs &a, const int32_t *thr) {
  if (!fp4_applies(a) || bd_applies(a) || fp6_applies(a)) return false;
  const int64_t nch = (int64_t)a.in.groups * a.cout;
  const float *f32c = (const float *)((const RqConst *)thr + 2 * (nch + 1));
  int32_t ok = 0;
  if (hipMemcpy(&ok, f32c + 3 * nch, sizeof(ok), hipMemcpyDeviceToHost) != hipSuccess) return false;
  return ok == 1;
}

int conv_mfma_epilogue(const ConvArgs &a, const int32_t *thr) {
  if (!bd_applies(a) && ((a.out.bits == 3 && !fp6_applies(a)) || (a.res.data && a.res.bits != 2))) return 1;
  int32_t flag = 0;
  const RqConst *rq = (const RqConst *)thr;
  if (hipMemcpy(&flag, rq + (int64_t)a.in.groups * a.cout, sizeof(flag), hipMemcpyDeviceToHost) != hipSuccess)
    return -1;
  return flag != 0 ? 1 : 0;
}

// Compute units of the current device (cached per device).
int cu_count() {
  static std::mutex mu;
  static int devs[16], vals[16], used = 0;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  std::lock_guard<std::mutex> lock(mu);
  for (int i = 0; i < used; ++i)
    if (devs[i] == dev) return vals[i];
  int cus = 256;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1) cus = 256;
  if (used < 16) {
    devs[used] = dev;
    vals[used] = cus;
    ++used;
  }
  return cus;
}

// Persistent workgroups of a tiled-kernel build: as many as are resident at
// once (registers and LDS decide; the variants with and without a shortcut
// need about the same), a multiple of 8.
int tile_slots(const void *kern, int threads) {
  // cached per kernel and device (a few dozen builds)
  static std::mutex mu;
  static const void *keys[64];
  static int devs[64], vals[64], used = 0;
  int dev = 0;
  hipGetDevice(&dev);
  std::lock_guard<std::mutex> lock(mu);
  for (int i = 0; i < used; ++i)
    if (keys[i] == kern && devs[i] == dev) return vals[i];
  int cus = 256, per = 2;
  hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, kern, threads, 0) != hipSuccess || per < 1) per = 1;
  const int v = std::max(8, cus * per / 8 * 8);
  if (used < 64) {
    keys[used] = kern;
    devs[used] = dev;
    vals[used] = v;
    ++used;
  }
  return v;
}

// The tiled kernel takes 2-bit grouped layers with 64-channel blocks and
// 2-bit outputs (and 2-bit or no identity shortcut); a layer whose requant
// needs the int64 path runs on the general partner launched beside it.
// 2-bit grouped layers with 2-bit outputs (and shortcut codes) and 64-channel
// blocks: the layers the tiled 2-bit builds take.
static bool grouped2_tiles(const ConvArgs &a) {
  const int64_t wbytes = (int64_t)a.in.groups * a.cout * make_geo(a).kb_total * 64;
  return !is_stem(a) && a.in.bits == 2 && a.w_bits == 2 && a.cout % 64 == 0 && wbytes < ((int64_t)1 << 30) &&
         a.out.bits == 2 && (!a.res.data || a.res.bits == 2);
}

// The persistent int8 tile kernel keeps its ring full across tiles: at least
// kStages K-blocks per tile.
bool tile_kernel_applies(const ConvArgs &a) { return grouped2_tiles(a) && make_geo(a).kb_total >= kStages; }

// FP4 matrix cores for a 2-bit tiled layer whose accumulator bound is below
// 2^23 (the fp32 accumulator then holds every partial sum, and the shortcut
// term, exactly), unless the context keeps layers on int8 (a.fp4 = 0).  The
// FP4 kernel runs one tile per workgroup and takes any K-block count (1 x 1
// layers over 64 or 128 input channels included).
bool fp4_applies(const ConvArgs &a) { return a.fp4 && grouped2_tiles(a) && acc_bound_of(a) < ((int64_t)1 << 23); }

// FP6 matrix cores for 3-bit grouped layers with 3-bit outputs, 64-channel
// blocks and no shortcut, under the same accumulator bound (the fp32
// accumulator holds t / 8: a multiple of 1/8 below 2^20 is exact) and the
// same context switch.
bool fp6_applies(const ConvArgs &a) {
  const int64_t wbytes = (int64_t)a.in.groups * a.cout * make_geo(a).kb_total * 64;
  return a.fp4 && !is_stem(a) && a.in.bits == 3 && a.w_bits == 3 && a.out.bits == 3 && !a.in.is_signed &&
         !a.res.data && !a.proj.data && a.cout % 64 == 0 && a.in.cpg % 64 == 0 && wbytes < ((int64_t)1 << 30) &&
         acc_bound_of(a) < ((int64_t)1 << 23);
}

// The Eq. 4 bit decomposition (palq_set_conv_bitdecomp) for an unsigned
// M-bit layer (M in {4, 6, 8}) with M-bit weights, outputs and shortcut
// codes and 64-channel blocks, when each fp32 accumulator stays exact: its
// bound K sum 4^(i+j-base) max|x_i| max|w_j| over the chunk pairs it takes
// (x_i <= 3, w_j <= 3 or, the top chunk, 2 in magnitude) is below 2^24.
bool bd_applies(const ConvArgs &a) {
  const int M = a.in.bits, GC = M / 2;
  if (!a.bitdecomp || is_stem(a) || a.in.is_signed || (M != 4 && M != 6 && M != 8) || a.w_bits != M ||
      a.out.bits != M || a.in.cpg % 64 != 0 || a.cout % 64 != 0)
    return false;
  if (a.res.data && (a.res.bits != M || a.res.is_signed)) return false;
  if (a.proj.data && (a.proj.bits != M || a.proj.cpg % 64 != 0 || a.proj.is_signed)) return false;
  if ((int64_t)a.in.groups * a.cout * make_geo(a).kb_total * GC * 32 >= ((int64_t)1 << 30)) return false;
  const int64_t K = (int64_t)a.kh * a.kw * a.in.cpg + (a.proj.data ? a.proj.cpg : 0);
  int64_t lo = 0, hi = 0;
  for (int i = 0; i < GC; ++i)
    for (int j = 0; j < GC; ++j) {
      const int64_t term = ((int64_t)1 << (2 * (i + j))) * 3 * (j == GC - 1 ? 2 : 3);
      if (M == 8 && i + j >= 3) hi += term >> 6;
      else lo += term;
    }
  return K * lo < ((int64_t)1 << 24) && K * hi < ((int64_t)1 << 24);
}
// The decomposition's weight slabs follow the int8 slabs (and Geo::acc0).
size_t bd_offset(const ConvArgs &a) {
  const size_t nch = (size_t)a.in.groups * a.cout;
  return (nch * make_geo(a).kb_total * 64 + (a.in.bits >= 6 ? nch * 4 : 0) + 255) & ~(size_t)255;
}

// The stem on the tiled kernel: explicit zero border (pad 0), 128-channel
// blocks, no shortcut, no accumulator dump.
bool stem_tile_applies(const ConvArgs &a) {
  return is_stem(a) && a.pad == 0 && a.cout % 128 == 0 && !a.res.data && !a.acc_dump && a.out.bits == 2 &&
         (int64_t)a.in.groups * a.cout * make_geo(a).kb_total * 64 < ((int64_t)1 << 30);
}

// Stems whose weights are also prepacked by filter row (prepack_stem_rows_kernel,
// after the K-block slabs): one input group, 7 filter rows of at most 8 taps,
// stride 2.
bool stem_rows(const ConvArgs &a) {
  return stem_tile_applies(a) && a.in.groups == 1 && a.kh == sp::KH && a.kw <= 8 && a.stride == 2;
}
size_t stem_rows_offset(const ConvArgs &a) { return (size_t)a.in.groups * a.cout * make_geo(a).kb_total * 64; }

// Tiled-kernel builds (tile shape per wave CB x PB blocks of 32 x 32, WN x WM
// waves): the 8-bit stem; 2-bit layers on FP4 with 64-channel blocks (1 x 4
// waves, 256-pixel tiles), 128-channel blocks (2 x 2 waves, 128 pixels) or
// 128-channel blocks with 2 x 4 blocks per wave (256 pixels); 2-bit layers on
// int8 with 64- or 128-channel blocks (256 pixels).
// 3-bit layers on FP6 with 64-channel (1 x 4 waves, 256 pixels) or
// 128-channel blocks (2 x 2 waves, 128 pixels).
// Wide layers as the Eq. 4 decomposition with 64- or 128-channel tiles.
enum TileBuild {
  kTileNone = 0, kTileStem, kTileFp4C64, kTileFp4C128, kTileFp4C128P4, kTileFp4C128K2, kTileFp6C64, kTileFp6C128,
  kTileI8C64, kTileI8C128, kTileBdC64, kTileBdC128
};

// 2 x 4 blocks per wave (256-pixel tiles) for 128-channel FP4 layers where
// the bigger tiles leave every CU at least one and do not lengthen the
// busiest CU's share: 2 ceil(T4 / CUs) <= ceil(T2 / CUs) tile units.
bool fp4_pb4_pays(const ConvArgs &a, const Geo &geo) {
  const int64_t m = geo.M, tiles_per_px = (int64_t)(a.cout / 128) * a.in.groups;
  const int64_t t2 = (m + 127) / 128 * tiles_per_px, t4 = (m + 255) / 256 * tiles_per_px;
  const int64_t cus = cu_count();
  return t4 >= cus && 2 * ((t4 + cus - 1) / cus) <= (t2 + cus - 1) / cus;
}

// The in-workgroup K split (conv_fpx_tile, KS = 2) for 128-channel FP4
// layers with fewer 128 x 128 tiles than twice the CUs (the deep layers,
// whose tiles leave most SIMDs with one wave): an even number of K-blocks
// per tap, an even projection and at least 8 K-blocks.
bool fp4_ksplit_pays(const ConvArgs &a, const Geo &geo) {
  const int64_t t2 = (geo.M + 127) / 128 * (a.cout / 128) * a.in.groups;
  const int pk = geo.kb_total - geo.kb_main;
  return geo.cpb % 2 == 0 && pk % 2 == 0 && geo.kb_total >= 8 && t2 < 2 * (int64_t)cu_count();
}

// The one selection rule of the conv launches: which tiled build (if any)
// takes the layer given the epilogue build epi (0 fast, 1 general, -1 not
// known: a tiled build is then launched with its general partner, which
// runs only if the layer's int64-requant flag is set).
struct ConvChoice {
  int tile;  // TileBuild
  int cb;    // channel blocks of the persistent build (0: it does not fit LDS)
};

ConvChoice conv_choice(const ConvArgs &a, const Geo &geo, int epi) {
  ConvChoice c{kTileNone, pick_cb(a, geo)};
  if (epi == 1) return c;
  if (bd_applies(a)) {
    c.tile = a.cout % 128 ? kTileBdC64 : kTileBdC128;
    return c;
  }
  if (fp6_applies(a)) {
    c.tile = a.cout % 128 ? kTileFp6C64 : kTileFp6C128;
    return c;
  }
  if (a.out.bits == 3) return c;
  if (stem_tile_applies(a)) c.tile = kTileStem;
  else if (fp4_applies(a))
    c.tile = a.cout % 128             ? kTileFp4C64
             : fp4_pb4_pays(a, geo)    ? kTileFp4C128P4
             : fp4_ksplit_pays(a, geo) ? kTileFp4C128K2
                                       : kTileFp4C128;
  else if (tile_kernel_applies(a)) c.tile = a.cout % 128 ? kTileI8C64 : kTileI8C128;
  return c;
}

// The FP4 grouped kernel: one workgroup per tile, XCD-contiguous runs of the
// chunked tile order (32 chunks where the packed input outweighs the filter,
// as in launch_tile).
template <int B, int CB, int PB, int WN, int WM, int KS = 1>
hipError_t launch_fpx(const ConvArgs &a, const Geo &geo, hipStream_t s) {
  constexpr int S = 4;
  using C = f4::Cfg<CB, PB, WN, WM, B>;
  const int npt = (int)((geo.M + C::TM - 1) / C::TM);
  const int ncb = a.cout / C::TN;
  const int64_t T = (int64_t)npt * ncb * a.in.groups;
  if (T <= 0 || T > 0x3fffffff || geo.kb_total < 1) return hipErrorInvalidValue;
  const int64_t wbytes = (int64_t)a.in.groups * a.cout * geo.kb_total * (C::SLAB / 32);
  const int64_t xbytes = a.in.bytes;
  const int nch = 7 * wbytes < (int64_t)(a.in.groups - 1) * xbytes ? std::min(32, npt) : 1;
  if (KS == 2 && (geo.kb_total % 2 != 0 || geo.cpb % 2 != 0)) return hipErrorInvalidValue;
  const dim3 grid((unsigned)((T + 7) / 8 * 8)), block(C::NT * KS);
  if constexpr (B == 3) {
    if (a.res.data || a.proj.data) return hipErrorNotSupported;
    if (!a.acc_dump)
      hipLaunchKernelGGL((conv_fp6_kernel<CB, PB, WN, WM, false, S>), grid, block, 0, s, a, geo, npt, ncb, nch);
    else
      hipLaunchKernelGGL((conv_fp6_kernel<CB, PB, WN, WM, true, S>), grid, block, 0, s, a, geo, npt, ncb, nch);
    return hipGetLastError();
  }
  // the fp32 requant where the plan found it exact for every channel
  if (a.f32ep) {
    if (!a.res.data && !a.acc_dump)
      hipLaunchKernelGGL((conv_fp4_kernel<CB, PB, WN, WM, 0, false, S, true, KS>), grid, block, 0, s, a, geo, npt, ncb, nch);
    else if (!a.acc_dump)
      hipLaunchKernelGGL((conv_fp4_kernel<CB, PB, WN, WM, 2, false, S, true, KS>), grid, block, 0, s, a, geo, npt, ncb, nch);
    else if (!a.res.data)
      hipLaunchKernelGGL((conv_fp4_kernel<CB, PB, WN, WM, 0, true, S, true, KS>), grid, block, 0, s, a, geo, npt, ncb, nch);
    else
      hipLaunchKernelGGL((conv_fp4_kernel<CB, PB, WN, WM, 2, true, S, true, KS>), grid, block, 0, s, a, geo, npt, ncb, nch);
    return hipGetLastError();
  }
  if (!a.res.data && !a.acc_dump)
    hipLaunchKernelGGL((conv_fp4_kernel<CB, PB, WN, WM, 0, false, S, false, KS>), grid, block, 0, s, a, geo, npt, ncb, nch);
  else if (!a.acc_dump)
    hipLaunchKernelGGL((conv_fp4_kernel<CB, PB, WN, WM, 2, false, S, false, KS>), grid, block, 0, s, a, geo, npt, ncb, nch);
  else if (!a.res.data)
    hipLaunchKernelGGL((conv_fp4_kernel<CB, PB, WN, WM, 0, true, S, false, KS>), grid, block, 0, s, a, geo, npt, ncb, nch);
  else
    hipLaunchKernelGGL((conv_fp4_kernel<CB, PB, WN, WM, 2, true, S, false, KS>), grid, block, 0, s, a, geo, npt, ncb, nch);
  return hipGetLastError();
}

// A tile kernel whose LDS is dynamic (lds bytes, above the static limit).
template <typename K>
hipError_t launch_dyn(K kern, const ConvArgs &a, const Geo &geo, dim3 grid, dim3 block, size_t lds, hipStream_t s,
                      int npt, int ncb, int nch) {
  hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, grid, block, lds, s, a, geo, npt, ncb, nch);
  return hipGetLastError();
}

// The Eq. 4 decomposition: as launch_fpx, with the ring in dynamic LDS.
template <int M, int WN>
hipError_t launch_bd(const ConvArgs &a, const Geo &geo, hipStream_t s) {
  using C = bd::Cfg<M, WN>;
  const int npt = (int)((geo.M + C::TM - 1) / C::TM);
  const int ncb = a.cout / C::TN;
  const int64_t T = (int64_t)npt * ncb * a.in.groups;
  if (T <= 0 || T > 0x3fffffff || geo.kb_total < 1) return hipErrorInvalidValue;
  const int64_t wbytes = (int64_t)a.in.groups * a.cout * geo.kb_total * C::GC * 32;
  const int64_t xbytes = a.in.bytes;
  const int nch = 7 * wbytes < (int64_t)(a.in.groups - 1) * xbytes ? std::min(32, npt) : 1;
  const size_t lds = (size_t)C::S * C::SST + (size_t)C::TN * (sizeof(RqConst) + 4);
  const dim3 grid((unsigned)((T + 7) / 8 * 8)), block(C::NT);
  if (a.res.data)
    return a.acc_dump ? launch_dyn(conv_bitdecomp_kernel<M, WN, -1, true>, a, geo, grid, block, lds, s, npt, ncb, nch)
                      : launch_dyn(conv_bitdecomp_kernel<M, WN, -1, false>, a, geo, grid, block, lds, s, npt, ncb, nch);
  return a.acc_dump ? launch_dyn(conv_bitdecomp_kernel<M, WN, 0, true>, a, geo, grid, block, lds, s, npt, ncb, nch)
                    : launch_dyn(conv_bitdecomp_kernel<M, WN, 0, false>, a, geo, grid, block, lds, s, npt, ncb, nch);
}

template <int M>
hipError_t launch_bd_m(const ConvArgs &a, const Geo &geo, int tile, hipStream_t s) {
  return tile == kTileBdC64 ? launch_bd<M, 1>(a, geo, s) : launch_bd<M, 2>(a, geo, s);
}

template <int CB, int PB, int WN, int WM, bool STEM = false, int S = PALQ_TILE_STAGES>
hipError_t launch_tile(const ConvArgs &a, const Geo &geo, hipStream_t s) {
  if (geo.kb_total < S) return hipErrorInvalidValue;
  constexpr int TN = WN * CB * 32, TM = WM * PB * 32;
  const int npt = (int)((geo.M + TM - 1) / TM);
  const int ncb = a.cout / TN;
  const int64_t T = (int64_t)npt * ncb * a.in.groups;
  if (T <= 0 || T > 0x7fffffff) return hipErrorInvalidValue;
  const int slots = tile_slots((const void *)conv_tile_kernel<CB, PB, WN, WM, STEM ? 0 : 2, STEM, S>, WN * WM * 64);
  // Pixel chunks (tile_at): 32 (four per XCD), so that an XCD fetches each
  // input line once for all groups while a chunk's lines still fit its L2,
  // unless the filter is the larger read (every XCD then reads all of it):
  // about 7 W extra against (G - 1) X saved.
  const int64_t wbytes = (int64_t)a.in.groups * a.cout * geo.kb_total * 64;
  const int64_t xbytes = a.in.bytes;
  const int nch = 7 * wbytes < (int64_t)(a.in.groups - 1) * xbytes ? std::min(32, npt) : 1;
  // P workgroups per XCD: all resident slots, no more than the XCD's
  // tiles, and runs of at most npt / nch tiles (two (chunk, combo) segments)
  const int64_t Tx = (T + 7) / 8;
  const int maxlen = npt / nch;
  int64_t P = std::max<int64_t>(1, std::min<int64_t>(slots / 8, Tx));
  if ((Tx + P - 1) / P > maxlen) P = (Tx + maxlen - 1) / maxlen;
  const dim3 grid((unsigned)(8 * P)), block(WN * WM * 64);
  if constexpr (STEM)
    hipLaunchKernelGGL((conv_tile_kernel<CB, PB, WN, WM, 0, true, S>), grid, block, 0, s, a, geo, npt, ncb, nch);
  else if (!a.res.data && !a.acc_dump)
    hipLaunchKernelGGL((conv_tile_kernel<CB, PB, WN, WM, 0, false, S>), grid, block, 0, s, a, geo, npt, ncb, nch);
  else if (!a.acc_dump)
    hipLaunchKernelGGL((conv_tile_kernel<CB, PB, WN, WM, 2, false, S>), grid, block, 0, s, a, geo, npt, ncb, nch);
  else if (!a.res.data)
    hipLaunchKernelGGL((conv_tile_kernel<CB, PB, WN, WM, 0, false, S, true>), grid, block, 0, s, a, geo, npt, ncb, nch);
  else
    hipLaunchKernelGGL((conv_tile_kernel<CB, PB, WN, WM, 2, false, S, true>), grid, block, 0, s, a, geo, npt, ncb, nch);
  return hipGetLastError();
}

// The stem followed by a 3x3 / stride 2 / pad 1 max pool of its output, on
// stem_pool_kernel: the stem's tiled-kernel conditions with a 7-row filter
// at stride 2 and its weights also prepacked by filter row (stem_rows), an
// input row of at most 1024 bytes (so at most 125 output columns), and a
// pooled view of the stem's output shape.  The caller must know the fast
// epilogue applies (conv_mfma_epilogue == 0): the kernel has no general
// build.
bool stem_pool_applies(const ConvArgs &a, const ActView &po, int k, int stride, int pad) {
  if (!stem_rows(a) || a.wo < 1 || a.ho < 1) return false;
  if (k != 3 || stride != 2 || pad != 1) return false;
  if (po.n != a.out.n || po.h != (a.ho + 1) / 2 || po.w != (a.wo + 1) / 2 || po.groups != a.out.groups ||
      po.cpg != a.out.cpg || po.bits != 2 || po.pixel != a.out.pixel || po.row != a.out.row ||
      po.gstride != po.row)  // the store offsets take a pixel's groups as adjacent rows
    return false;
  const int64_t in_bytes = a.in.bytes;
  const int64_t out_bytes = po.bytes;
  const int64_t units = (int64_t)a.out.n * (a.cout / 128) * po.h;
  return (int64_t)a.in.w * a.in.pixel <= sp::RB && in_bytes < 0x7fff0000 && out_bytes < 0x7fff0000 &&
         units < 0x7fffffff;
}

hipError_t launch_stem_pool(const ConvArgs &a, const uint8_t *wp, const int32_t *thr, const ActView &po,
                            hipStream_t s) {
  Geo geo = make_geo(a);
  if (geo.M == 0) return hipSuccess;
  geo.wp = wp;
  geo.rq = (const RqConst *)thr;
  const uint8_t *wrow = wp + stem_rows_offset(a);
  const int units = a.out.n * (a.cout / 128) * po.h;
  const int slots = tile_slots((const void *)stem_pool_kernel, sp::NT);
  // P workgroups per XCD: all resident slots, no more than the XCD's units,
  // and runs of at most ho2 units (two channel blocks' constants)
  const int64_t Tx = (units + 7) / 8;
  int64_t P = std::max<int64_t>(1, std::min<int64_t>(slots / 8, Tx));
  if ((Tx + P - 1) / P > po.h) P = (Tx + po.h - 1) / po.h;
  hipLaunchKernelGGL(stem_pool_kernel, dim3((unsigned)(8 * P)), dim3(sp::NT), 0, s, a, geo, po, wrow, units);
  return hipGetLastError();
}

const char *conv_kernel_label(const ConvArgs &a, int epi) {
  const Geo geo = make_geo(a);
  switch (conv_choice(a, geo, epi).tile) {
    case kTileStem: return "conv_tile_kernel[stem]";
    case kTileFp4C64: case kTileFp4C128: case kTileFp4C128P4: case kTileFp4C128K2: return "conv_fp4_kernel";
    case kTileFp6C64: case kTileFp6C128: return "conv_fp6_kernel";
    case kTileBdC64: case kTileBdC128: return "conv_bitdecomp_kernel";
    case kTileI8C64: case kTileI8C128: return "conv_tile_kernel[int8]";
    default: return is_stem(a) ? "conv_stem_kernel" : "conv_grouped_kernel";
  }
}

hipError_t launch_conv_mfma(const ConvArgs &a_in, const uint8_t *wp, const int32_t *thr, int epi, hipStream_t s) {
  ConvArgs a = a_in;
  a.gated = 0;
  Geo geo = make_geo(a);
  if (geo.M == 0) return hipSuccess;
  geo.wp = wp;
  geo.rq = (const RqConst *)thr;
  const ConvChoice c = conv_choice(a, geo, epi);
  if (c.cb == 0 && c.tile == kTileNone) return hipErrorNotSupported;  // no build for this layer
  if (a.acc_dump && c.tile == kTileNone) epi = 1;  // only the general persistent build dumps
  hipError_t e = hipSuccess;
  const int nch = a.in.groups * a.cout;
  Geo g4 = geo;  // FP4 (FP6) slabs and constants follow the int8 ones
  g4.wp = wp + (size_t)nch * geo.kb_total * 64;
  g4.rq = geo.rq + nch + 1;
  constexpr int S4 = PALQ_TILE_STAGES;
  switch (c.tile) {
    case kTileStem: e = launch_tile<2, 2, 2, 2, true, PALQ_STEM_STAGES>(a, geo, s); break;
    case kTileFp4C64: e = launch_fpx<2, 2, 2, 1, 4>(a, g4, s); break;
    case kTileFp4C128: e = launch_fpx<2, 2, 2, 2, 2>(a, g4, s); break;
    case kTileFp4C128P4: e = launch_fpx<2, 2, 4, 2, 2>(a, g4, s); break;
    case kTileFp4C128K2: e = launch_fpx<2, 2, 2, 2, 2, 2>(a, g4, s); break;
    case kTileFp6C64: e = launch_fpx<3, 2, 2, 1, 4>(a, g4, s); break;
    case kTileBdC64: case kTileBdC128: {
      Geo gb = g4;
      gb.wp = wp + bd_offset(a);
      e = a.in.bits == 4 ? launch_bd_m<4>(a, gb, c.tile, s)
                         : a.in.bits == 6 ? launch_bd_m<6>(a, gb, c.tile, s) : launch_bd_m<8>(a, gb, c.tile, s);
      break;
    }
    case kTileFp6C128: e = launch_fpx<3, 2, 2, 2, 2>(a, g4, s); break;
    case kTileI8C64: e = launch_tile<2, 2, 1, 4>(a, geo, s); break;
    case kTileI8C128: e = launch_tile<2, 2, 2, 4>(a, geo, s); break;
    default: break;
  }
  if (e != hipSuccess) return e;
  if (c.tile != kTileNone) {
    if (epi == 0) return hipSuccess;
    // epi unknown: the general partner, which runs only if the flag is set
    a.gated = 1;
    if (c.cb == 0) return launch_conv_direct(a, s, (const int32_t *)(geo.rq + nch));
    epi = 1;
  }
  const int cb = c.cb, pb = 1;
  if (is_stem(a)) return cb == 2 ? launch_stem<2, 1>(a, geo, epi, s) : launch_stem<1, 1>(a, geo, epi, s);
  switch (a.in.bits) {
    case 2: return dispatch_bits<2>(a, geo, cb, pb, epi, s);
    case 3: return dispatch_bits<3>(a, geo, cb, pb, epi, s);
    case 4: return dispatch_bits<4>(a, geo, cb, pb, epi, s);
    case 6: case 8:
      geo.acc0 = (const int32_t *)(wp + (size_t)nch * geo.kb_total * 64);
      return dispatch_bits<8>(a, geo, cb, pb, epi, s);
  }
  return hipErrorNotSupported;
}

// ---------------------------------------------------------------- static scratch
// palq_group_conv_noalloc's prepacked filter and requant constants: a
// file-scope device array, one copy on every GPU that loads the library
// (held until the process ends).  In host code `scratch` is only a handle
// for the runtime; kernels receive the device address that
// hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) uint8_t scratch[PALQ_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
uint8_t *g_scratch_ptr[kMaxScratchDevices];
bool g_scratch_looked_up[kMaxScratchDevices];
}  // namespace

hipError_t noalloc_scratch_init(int device) {
  if (device < 0 || device >= kMaxScratchDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_looked_up[device]) return g_scratch_ptr[device] ? hipSuccess : hipErrorInvalidSymbol;
  void *p = nullptr;
  const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  g_scratch_looked_up[device] = true;
  g_scratch_ptr[device] = (e == hipSuccess && p) ? (uint8_t *)p : nullptr;
  return e;
}

uint8_t *noalloc_scratch(int device) {
  if (device < 0 || device >= kMaxScratchDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  return g_scratch_ptr[device];
}

}  // namespace palq
