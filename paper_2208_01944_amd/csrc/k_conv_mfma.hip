// Grouped B-bit convolution as an implicit GEMM on gfx950 int8 MFMA.
//
// Per group g (Section 4.1: G independent B-bit convolutions) the layer is
// D[k][m] = sum_K W[k][K] X[K][m] (Eq. 1) with k an output channel of the
// group, m an output pixel (n, oy, ox) and K = (ky, kx, c).  One workgroup
// owns a tile of CB*32 output channels x 4*PB*32 pixels of one group; its
// four waves share the channels and split the pixels.
//
//  * Weights (MFMA A operand, rows = channels): packed b-bit units are read
//    from global memory, sign-extended to int8 in registers and written to
//    LDS in MFMA operand order, KS 64-code K-blocks per stage, two stages in
//    flight (one barrier per stage).
//  * Activations (MFMA B operand, columns = pixels): each lane reads its own
//    pixel's packed codes for the current tap straight from global memory
//    (the 3x3 taps re-hit L1/L2) and unpacks them in registers with a few
//    shift/mask operations.  K order inside a 16-code unit is permuted by
//    the unpack; the weights are placed with the same permutation, which
//    leaves the contraction unchanged.
//  * 2-bit codes: the unpack leaves code 4e+d of a unit at bits 2d..2d+1 of
//    byte e without shifting it down (d = 0, 1, 2) or after one shift
//    (d = 3), i.e. scaled by 1, 4, 16, 16; the weights of those positions
//    are pre-scaled by 16, 4, 1, 1 so every product carries the factor 16,
//    which the epilogue removes exactly with an arithmetic shift.
//  * Epilogue: int32 accumulator -> + bias + shortcut (int64) -> fixed-point
//    requant with ReLU -> b-bit codes, written to group (g + s) mod G: the
//    cyclic permutation of Eq. 8 is only the store address.  A projection
//    shortcut is fused as extra K-blocks (1x1 conv of the block input of the
//    destination group), so its accumulator lands in the same registers.
#include "codes.h"
#include "palq_internal.h"

namespace palq {

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * 64;

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
// codes, hi = the chunk's bit-2 word (bit 8e + 4j + d for code 4e + d).
__device__ inline v4i unpack3(uint32_t lo, uint32_t hi, int j) {
  v4i r;
  _Pragma("unroll") for (int d = 0; d < 4; ++d) {
    const uint32_t l2 = (lo >> (2 * d)) & 0x03030303u;
    const uint32_t h1 = (hi >> (4 * j + d)) & 0x01010101u;
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

// Raw packed words a lane holds for one K-block (its half: two units).
template <int B> struct Raw { uint32_t w[B]; };

template <int B>
__device__ inline Raw<B> load_half(const uint8_t *p, bool valid) {
  Raw<B> r;
  if constexpr (B == 2) {
    uint2 v = valid ? *(const uint2 *)p : make_uint2(0, 0);
    r.w[0] = v.x; r.w[1] = v.y;
  } else if constexpr (B == 4) {
    uint4 v = valid ? *(const uint4 *)p : make_uint4(0, 0, 0, 0);
    r.w[0] = v.x; r.w[1] = v.y; r.w[2] = v.z; r.w[3] = v.w;
  } else {
    const uint32_t *q = (const uint32_t *)p;
    r.w[0] = valid ? q[0] : 0u; r.w[1] = valid ? q[1] : 0u; r.w[2] = valid ? q[2] : 0u;
  }
  return r;
}

// MFMA B operand for K-step j (0/1) from a lane's raw half block.
template <int B>
__device__ inline v4i act_operand(const Raw<B> &r, int j) {
  if constexpr (B == 2) return act_unpack2(r.w[j]);
  else if constexpr (B == 4) return unpack4_nibbles(r.w[2 * j], r.w[2 * j + 1]);
  else return unpack3(r.w[j], r.w[2], j);
}

// Weight unit u (0..3) of a 64-code K-block starting at p -> operand.
template <int B>
__device__ inline v4i load_weight_unit(const uint8_t *p, int u) {
  const uint32_t *q = (const uint32_t *)p;
  if constexpr (B == 2) return wt_unpack2(q[u]);
  else if constexpr (B == 4) return wt_unpack4(q[2 * u], q[2 * u + 1]);
  else return wt_unpack3(q[3 * (u >> 1) + (u & 1)], q[3 * (u >> 1) + 2], u & 1);
}

// ---------------------------------------------------------------- epilogue
__device__ inline int64_t requant_one(int64_t t, int32_t m, int32_t sh, int qmax) {
  const int64_t num = t * (int64_t)m + ((int64_t)1 << (sh - 1));
  int64_t q = num >> sh;
  q = q < 0 ? 0 : q;
  return q > qmax ? qmax : q;
}

// Code j (0..31) of a 32-code chunk held in registers.
__device__ inline int chunk_code(const uint32_t *cw, int j, int bits) {
  if (bits == 3) {
    uint32_t v = (cw[j >> 4] >> (2 * (j & 15))) & 3u;
    return (int)(v | (((cw[2] >> b3_hi_pos(j)) & 1u) << 2));
  }
  const int bit = j * bits;
  return (int)((cw[bit >> 5] >> (bit & 31)) & ((1u << bits) - 1u));
}

// ---------------------------------------------------------------- kernel
struct Geo {
  int32_t M;          // output pixels per group
  int32_t taps;       // kh * kw
  int32_t cpb;        // 64-code blocks per tap row
  int32_t kb_main;    // taps * cpb
  int32_t kb_total;   // + projection blocks
  int32_t pcpb;       // projection 64-code blocks
  int64_t w_ch;       // bytes of one output channel's filter (all taps)
  int64_t pw_ch;      // bytes of one projection channel
};

template <int B, int CB, int PB, int KS>
__global__ __launch_bounds__(kThreads) void conv_mfma_kernel(ConvArgs a, Geo geo) {
  constexpr int TPIX = kWaves * PB * 32;
  constexpr int KSTEP_BYTES = 32 * 16;                 // one (cb, half) slab: 32 ch x 16 B
  constexpr int KBLK_BYTES = 2 * CB * 2 * KSTEP_BYTES; // 2 K-steps x CB x 2 halves
  constexpr int STAGE_BYTES = KS * KBLK_BYTES;
  __shared__ __attribute__((aligned(16))) uint8_t lds[2 * STAGE_BYTES];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int l32 = lane & 31;
  const int half = lane >> 5;

  const int G = a.in.groups;
  const int g = blockIdx.z;
  const int gd = (g + a.shuffle) % G;
  const int ch0 = blockIdx.y * CB * 32;          // first output channel of the tile (in group)
  const int64_t m0 = (int64_t)blockIdx.x * TPIX;

  // ---- per pixel-block geometry of this lane
  int iy0[PB], ix0[PB], nimg[PB];
  bool pvalid[PB];
  int64_t mpix[PB];
  _Pragma("unroll") for (int pb = 0; pb < PB; ++pb) {
    const int64_t m = m0 + (wave * PB + pb) * 32 + l32;
    mpix[pb] = m;
    pvalid[pb] = m < geo.M;
    const int64_t mm = pvalid[pb] ? m : 0;
    const int ox = (int)(mm % a.wo);
    const int oy = (int)((mm / a.wo) % a.ho);
    nimg[pb] = (int)(mm / ((int64_t)a.wo * a.ho));
    iy0[pb] = oy * a.stride - a.pad;
    ix0[pb] = ox * a.stride - a.pad;
  }

  // ---- weight staging: items (cb, ch, kbl, u), 4 units per (channel, block)
  constexpr int ITEMS = CB * 32 * KS * 4;
  static_assert(ITEMS % kThreads == 0, "stage items must divide the block");
  constexpr int IPT = ITEMS / kThreads;

  auto stage_weights = [&](int kb0, v4i (&regs)[IPT]) {
    _Pragma("unroll") for (int i = 0; i < IPT; ++i) {
      const int item = i * kThreads + tid;
      const int u = item & 3;
      const int kbl = (item >> 2) % KS;
      const int chn = (item >> 2) / KS;  // cb*32 + ch
      const int kb = kb0 + kbl;
      v4i v = {0, 0, 0, 0};
      if (kb < geo.kb_total) {
        const int k = ch0 + chn;
        const uint8_t *p;
        if (kb < geo.kb_main) {
          p = a.w + ((int64_t)g * a.cout + k) * geo.w_ch + (int64_t)kb * Blk<B>::bytes;
        } else {
          p = a.proj_w + ((int64_t)gd * a.cout + k) * geo.pw_ch +
              (int64_t)(kb - geo.kb_main) * Blk<B>::bytes;
        }
        v = load_weight_unit<B>(p, u);
      }
      regs[i] = v;
    }
  };
  auto store_weights = [&](int buf, const v4i (&regs)[IPT]) {
    _Pragma("unroll") for (int i = 0; i < IPT; ++i) {
      const int item = i * kThreads + tid;
      const int u = item & 3;
      const int kbl = (item >> 2) % KS;
      const int chn = (item >> 2) / KS;
      const int cb = chn >> 5, ch = chn & 31;
      const int h = u >> 1, j = u & 1;
      const int off = buf * STAGE_BYTES + kbl * KBLK_BYTES + ((j * CB + cb) * 2 + h) * KSTEP_BYTES +
                      ch * 16;
      *(v4i *)(lds + off) = regs[i];
    }
  };

  // ---- activation addressing for K-block kb
  const int64_t in_img = (int64_t)a.in.h * a.in.w;
  auto act_ptr = [&](int kb, int pb, bool &valid) -> const uint8_t * {
    if (kb < geo.kb_main) {
      const int tap = kb / geo.cpb;
      const int cblk = kb - tap * geo.cpb;
      const int ky = tap / a.kw, kx = tap - (tap / a.kw) * a.kw;
      const int iy = iy0[pb] + ky, ix = ix0[pb] + kx;
      valid = pvalid[pb] && iy >= 0 && iy < a.in.h && ix >= 0 && ix < a.in.w;
      const int64_t pix = (int64_t)nimg[pb] * in_img + (int64_t)(valid ? iy : 0) * a.in.w + (valid ? ix : 0);
      return a.in.data + pix * a.in.pixel + (int64_t)g * a.in.row + cblk * Blk<B>::bytes +
             half * (Blk<B>::bytes / 2);
    }
    const int cblk = kb - geo.kb_main;
    const int iy = (iy0[pb] + a.pad) * a.proj_stride / a.stride;
    const int ix = (ix0[pb] + a.pad) * a.proj_stride / a.stride;
    valid = pvalid[pb];
    const int64_t pix = ((int64_t)nimg[pb] * a.proj.h + iy) * a.proj.w + ix;
    return a.proj.data + pix * a.proj.pixel + (int64_t)gd * a.proj.row + cblk * Blk<B>::bytes +
           half * (Blk<B>::bytes / 2);
  };

  v16i acc[CB][PB];
  _Pragma("unroll") for (int cb = 0; cb < CB; ++cb)
    _Pragma("unroll") for (int pb = 0; pb < PB; ++pb)
      _Pragma("unroll") for (int r = 0; r < 16; ++r) acc[cb][pb][r] = 0;

  const int nstages = (geo.kb_total + KS - 1) / KS;
  v4i wreg[IPT];
  stage_weights(0, wreg);
  store_weights(0, wreg);
  __syncthreads();

  Raw<B> xcur[PB];
  _Pragma("unroll") for (int pb = 0; pb < PB; ++pb) {
    bool v;
    const uint8_t *p = act_ptr(0, pb, v);
    xcur[pb] = load_half<B>(p, v);
  }

  for (int s = 0; s < nstages; ++s) {
    const int buf = s & 1;
    if (s + 1 < nstages) stage_weights((s + 1) * KS, wreg);
    const int kb0 = s * KS;
    const int kmax = min(KS, geo.kb_total - kb0);
    for (int kbl = 0; kbl < kmax; ++kbl) {
      const int kb = kb0 + kbl;
      // prefetch the next K-block's activations
      Raw<B> xnext[PB];
      if (kb + 1 < geo.kb_total) {
        _Pragma("unroll") for (int pb = 0; pb < PB; ++pb) {
          bool v;
          const uint8_t *p = act_ptr(kb + 1, pb, v);
          xnext[pb] = load_half<B>(p, v);
        }
      }
      _Pragma("unroll") for (int j = 0; j < 2; ++j) {
        v4i bop[PB];
        _Pragma("unroll") for (int pb = 0; pb < PB; ++pb) bop[pb] = act_operand<B>(xcur[pb], j);
        _Pragma("unroll") for (int cb = 0; cb < CB; ++cb) {
          const v4i aop = *(const v4i *)(lds + buf * STAGE_BYTES + kbl * KBLK_BYTES +
                                         ((j * CB + cb) * 2 + half) * KSTEP_BYTES + l32 * 16);
          _Pragma("unroll") for (int pb = 0; pb < PB; ++pb)
            acc[cb][pb] = __builtin_amdgcn_mfma_i32_32x32x32_i8(aop, bop[pb], acc[cb][pb], 0, 0, 0);
        }
      }
      if (kb + 1 < geo.kb_total)
        _Pragma("unroll") for (int pb = 0; pb < PB; ++pb) xcur[pb] = xnext[pb];
    }
    if (s + 1 < nstages) store_weights(buf ^ 1, wreg);
    __syncthreads();
  }

  // ---------------------------------------------------------------- epilogue
  // Lane holds, for block (cb, pb), rows (channels) 8*(r/4) + 4*half + r%4 of
  // pixel l32: four quads Q = 2*qi + half of four consecutive channels.
  const int qmax = (1 << a.out.bits) - 1;
  const int bo = a.out.bits;
  const int64_t outC = (int64_t)G * a.cout;
  _Pragma("unroll") for (int cb = 0; cb < CB; ++cb) {
    const int kc = ch0 + cb * 32;   // first channel of this 32-channel chunk (in group)
    const int csb = g * a.cout + kc;
    const int cdb = gd * a.cout + kc;
    // quad values per pixel block
    uint32_t qv[PB][4];
    uint32_t hq[PB][4];  // bit-2 nibbles for 3-bit output
    _Pragma("unroll") for (int qi = 0; qi < 4; ++qi) {
      const int cq = 8 * qi + 4 * half;  // first channel of this quad within the chunk
      const v4i mul = *(const v4i *)(a.mult + csb + cq);
      const v4i shf = *(const v4i *)(a.shift + csb + cq);
      v4i bia = {0, 0, 0, 0};
      if (a.bias) bia = *(const v4i *)(a.bias + csb + cq);
      v4i rmu = {0, 0, 0, 0};
      if (a.res.data) rmu = *(const v4i *)(a.res_mult + csb + cq);
      _Pragma("unroll") for (int pb = 0; pb < PB; ++pb) {
        uint32_t rw[8];
        if (a.res.data) {
          const int rb = a.res.bits;
          const int nw = rb == 3 ? 3 : rb;
          const uint32_t *rp = (const uint32_t *)(a.res.data + (pvalid[pb] ? mpix[pb] : 0) * a.res.pixel +
                                                  (int64_t)gd * a.res.row) +
                               (int64_t)(kc >> 5) * nw;
          _Pragma("unroll") for (int k = 0; k < 8; ++k) rw[k] = k < nw ? rp[k] : 0u;
        }
        uint32_t qword = 0, hword = 0;
        int32_t accq[4];
        _Pragma("unroll") for (int e = 0; e < 4; ++e) {
          int32_t av = acc[cb][pb][4 * qi + e];
          if (B == 2) av >>= 4;  // remove the x16 operand scale (exact)
          accq[e] = av;
          int64_t t = (int64_t)av + bia[e];
          if (a.res.data) t += (int64_t)rmu[e] * chunk_code(rw, cq + e, a.res.bits);
          const uint32_t q = (uint32_t)requant_one(t, mul[e], shf[e], qmax);
          if (bo == 3) {
            qword |= (q & 3u) << (2 * e);
            hword |= ((q >> 2) & 1u) << e;
          } else {
            qword |= q << (bo * e);
          }
        }
        qv[pb][qi] = qword;
        hq[pb][qi] = hword;
        if (a.acc_dump && pvalid[pb]) {
          v4i dv = {accq[0], accq[1], accq[2], accq[3]};
          *(v4i *)(a.acc_dump + mpix[pb] * outC + cdb + cq) = dv;
        }
      }
    }
    // exchange quads with the partner lane (half ^ 1) and store
    _Pragma("unroll") for (int pb = 0; pb < PB; ++pb) {
      const uint32_t s0 = half ? qv[pb][0] : qv[pb][2];
      const uint32_t s1 = half ? qv[pb][1] : qv[pb][3];
      const uint32_t r0 = (uint32_t)__shfl_xor((int)s0, 32);
      const uint32_t r1 = (uint32_t)__shfl_xor((int)s1, 32);
      // the four quads this lane writes, in channel order
      uint32_t Q[4];
      if (half == 0) { Q[0] = qv[pb][0]; Q[1] = r0; Q[2] = qv[pb][1]; Q[3] = r1; }
      else           { Q[0] = r0; Q[1] = qv[pb][2]; Q[2] = r1; Q[3] = qv[pb][3]; }
      uint32_t hpart = 0;
      if (bo == 3) {
        _Pragma("unroll") for (int qi = 0; qi < 4; ++qi) {
          const int Qn = 2 * qi + half;
          hpart |= hq[pb][qi] << (8 * (Qn & 3) + 4 * (Qn >> 2));
        }
        hpart |= (uint32_t)__shfl_xor((int)hpart, 32);
      }
      if (!pvalid[pb]) continue;
      uint8_t *orow = a.out.data + mpix[pb] * a.out.pixel + (int64_t)gd * a.out.row;
      if (bo == 3) {
        uint32_t *cw = (uint32_t *)orow + (int64_t)(kc >> 5) * 3;
        const uint32_t lo = Q[0] | (Q[1] << 8) | (Q[2] << 16) | (Q[3] << 24);
        cw[half] = lo;
        if (half == 0) cw[2] = hpart;
      } else {
        // 16*bo bits per lane: bo/2 words
        uint32_t *cw = (uint32_t *)orow + (int64_t)(kc >> 5) * bo + half * (bo / 2);
        if (bo == 2) {
          cw[0] = Q[0] | (Q[1] << 8) | (Q[2] << 16) | (Q[3] << 24);
        } else if (bo == 4) {
          cw[0] = Q[0] | (Q[1] << 16);
          cw[1] = Q[2] | (Q[3] << 16);
        } else {
          cw[0] = Q[0]; cw[1] = Q[1]; cw[2] = Q[2]; cw[3] = Q[3];
        }
      }
    }
  }
}

template <int B, int CB, int PB, int KS>
hipError_t launch_cfg(const ConvArgs &a, const Geo &geo, hipStream_t s) {
  constexpr int TPIX = kWaves * PB * 32;
  dim3 grid((unsigned)((geo.M + TPIX - 1) / TPIX), (unsigned)(a.cout / (CB * 32)),
            (unsigned)a.in.groups);
  hipLaunchKernelGGL((conv_mfma_kernel<B, CB, PB, KS>), grid, dim3(kThreads), 0, s, a, geo);
  return hipGetLastError();
}

template <int B>
hipError_t launch_bits(const ConvArgs &a, const Geo &geo, hipStream_t s) {
  const int cb = (a.cout % 64 == 0) ? 2 : 1;
  // smallest pixel tile that still gives about two workgroups per CU
  const int64_t ch_tiles = (int64_t)(a.cout / (cb * 32)) * a.in.groups;
  const int64_t want = 512;
  int pb = 4;
  while (pb > 1 && ((geo.M + kWaves * pb * 32 - 1) / (kWaves * pb * 32)) * ch_tiles < want) pb >>= 1;
  if (cb == 2) {
    if (pb == 4) return launch_cfg<B, 2, 4, 4>(a, geo, s);
    if (pb == 2) return launch_cfg<B, 2, 2, 4>(a, geo, s);
    return launch_cfg<B, 2, 1, 4>(a, geo, s);
  }
  if (pb == 4) return launch_cfg<B, 1, 4, 8>(a, geo, s);
  if (pb == 2) return launch_cfg<B, 1, 2, 8>(a, geo, s);
  return launch_cfg<B, 1, 1, 8>(a, geo, s);
}

}  // namespace

bool conv_mfma_supported(const ConvArgs &a) {
  const int b = a.in.bits;
  if (a.in.is_signed || (b != 2 && b != 3 && b != 4) || a.w_bits != b) return false;
  if (a.in.cpg % 64 != 0 || a.cout % 32 != 0) return false;
  if (a.proj.data && (a.proj.bits != b || a.proj.cpg % 64 != 0 || a.proj.is_signed)) return false;
  return true;
}

hipError_t launch_conv_mfma(const ConvArgs &a, hipStream_t s) {
  Geo geo;
  geo.M = a.out.n * a.ho * a.wo;
  geo.taps = a.kh * a.kw;
  geo.cpb = a.in.cpg / 64;
  geo.kb_main = geo.taps * geo.cpb;
  geo.pcpb = a.proj.data ? a.proj.cpg / 64 : 0;
  geo.kb_total = geo.kb_main + geo.pcpb;
  geo.w_ch = (int64_t)geo.taps * row_bytes(a.in.cpg, a.w_bits);
  geo.pw_ch = a.proj.data ? row_bytes(a.proj.cpg, a.w_bits) : 0;
  if (geo.M == 0) return hipSuccess;
  switch (a.in.bits) {
    case 2: return launch_bits<2>(a, geo, s);
    case 3: return launch_bits<3>(a, geo, s);
    case 4: return launch_bits<4>(a, geo, s);
  }
  return hipErrorNotSupported;
}

}  // namespace palq
