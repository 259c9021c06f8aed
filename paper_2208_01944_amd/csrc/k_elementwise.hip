// Element-wise and reduction kernels of the PalQuant path: pack/unpack,
// the Eq. 2 quantiser with its min/max calibration, the standalone cyclic
// permutation (Eq. 8), max pool, integer global sum and the FC layer.
// All are bandwidth-bound; one thread handles one 32-code chunk of a row so
// that every packed word is written by exactly one thread.
#include <float.h>
#include <math.h>

#include "codes.h"
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
  const int per_chunk = out.bits == 3 ? 3 : out.bits;
  const int nw = chunk_words_in_row(ci, out.bits, out.row / 4);
  uint32_t *dst = (uint32_t *)(out.data + r * out.row) + (int64_t)ci * per_chunk;
  for (int k = 0; k < nw; ++k) dst[k] = words[k];
}

__global__ void unpack_kernel(ActView in, uint8_t *codes, int64_t rows, int chunks) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= rows * chunks) return;
  const int64_t r = t / chunks;
  const int ci = (int)(t % chunks);
  const int j0 = ci * 32;
  const int nc = min(32, in.cpg - j0);
  const uint8_t *row = in.data + r * in.row;
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
  uint32_t *dst = (uint32_t *)(out.data + r * out.row);
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
  const int per = 32 / out.bits;
  const int j0 = wi * per;
  const int nc = min(per, out.cpg - j0);
  const uint32_t mask = (1u << out.bits) - 1u;
  uint32_t w = 0;
  for (int k = 0; k < nc; ++k) {
    const int q = (degenerate ? 0 : quant_one(src[j0 + k], l, rng, qmax)) - off;
    w |= ((uint32_t)q & mask) << (k * out.bits);
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
  const uint32_t *src = (const uint32_t *)(in.data + p * in.pixel + g * in.row);
  uint32_t *dst = (uint32_t *)(out.data + p * out.pixel + gd * out.row);
  dst[wi] = src[wi];
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
  uint32_t *dst = (uint32_t *)(out.data + r * out.row);
  if (in.bits == 2) {
    uint32_t m = 0;
    for (int ky = 0; ky < k; ++ky) {
      const int iy = oy * stride - pad + ky;
      if (iy < 0 || iy >= in.h) continue;
      for (int kx = 0; kx < k; ++kx) {
        const int ix = ox * stride - pad + kx;
        if (ix < 0 || ix >= in.w) continue;
        const uint32_t *row = (const uint32_t *)(in.data + (((int64_t)n * in.h + iy) * in.w + ix) * in.pixel +
                                                 (int64_t)g * in.row);
        m = max2x16(m, row[wi]);
      }
    }
    const int used = out.cpg * 2 - wi * 32;  // code bits of this word inside the row
    dst[wi] = used >= 32 ? m : (m & ((1u << used) - 1u));
    return;
  }
  const int per = in.bits == 3 ? 32 : 32 / in.bits;
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
      const uint8_t *row = in.data + (((int64_t)n * in.h + iy) * in.w + ix) * in.pixel + g * in.row;
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
    for (int j = 0; j < nc; ++j) w |= (uint32_t)c[j] << (j * in.bits);
    dst[wi] = w;
  }
}

// ------------------------------------------------------------ global sum
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
    s += read_code(in.data + ((int64_t)n * hw + p) * in.pixel + g * in.row, j, in.bits, 0);
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

}  // namespace

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

hipError_t launch_quantize(const float *x, float l, float u, const float *range, const ActView &out,
                           hipStream_t s) {
  const int64_t rows = (int64_t)out.n * out.h * out.w * out.groups;
  const int units = out.bits == 3 ? (out.cpg + 31) / 32 : (int)(out.row / 4);
  if (rows == 0) return hipSuccess;
  hipLaunchKernelGGL(quantize_kernel, dim3(grid_for(rows * units)), dim3(kBlock), 0, s, x, l, u,
                     (const uint32_t *)range, out, rows, units);
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

hipError_t launch_maxpool(const ActView &in, int k, int stride, int pad, const ActView &out,
                          hipStream_t s) {
  const int64_t rows = (int64_t)out.n * out.h * out.w * out.groups;
  const int units = out.bits == 3 ? (out.cpg + 31) / 32 : (int)(out.row / 4);
  if (rows == 0) return hipSuccess;
  hipLaunchKernelGGL(maxpool_kernel, dim3(grid_for(rows * units)), dim3(kBlock), 0, s, in, k,
                     stride, pad, out, units);
  return hipGetLastError();
}

hipError_t launch_avgsum(const ActView &in, int32_t *out, hipStream_t s) {
  const int64_t items = (int64_t)in.n * in.groups * in.cpg;
  if (items == 0) return hipSuccess;
  hipLaunchKernelGGL(avgsum_kernel, dim3(grid_for(items)), dim3(kBlock), 0, s, in, out);
  return hipGetLastError();
}

hipError_t launch_fc(const int32_t *x, int n, int cin, const int8_t *w, int cout, int32_t *logits,
                     hipStream_t s) {
  const int64_t items = (int64_t)n * cout;
  if (items == 0) return hipSuccess;
  hipLaunchKernelGGL(fill_i32_kernel, dim3(grid_for(items)), dim3(kBlock), 0, s, logits, items);
  dim3 grid((unsigned)((cout + FC_T - 1) / FC_T), (unsigned)((n + FC_T - 1) / FC_T),
            (unsigned)((cin + FC_KS - 1) / FC_KS));
  hipLaunchKernelGGL(fc_kernel, grid, dim3(256), 0, s, x, n, cin, w, cout, logits);
  return hipGetLastError();
}

}  // namespace palq
