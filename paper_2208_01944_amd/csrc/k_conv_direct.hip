// Direct grouped convolution: one thread per (output pixel, destination
// group, 32-code output chunk), scalar integer multiply-accumulate.  It
// covers every shape and bit width the ABI accepts (odd channel counts,
// mixed activation/weight widths) and is the path for layers the MFMA
// kernel does not take.  Same epilogue arithmetic as the MFMA kernel.
#include "codes.h"
#include "palq_internal.h"

namespace palq {

namespace {

__device__ inline int64_t requant_one(int64_t t, int32_t m, int32_t sh, int qmax) {
  const int64_t num = t * (int64_t)m + ((int64_t)1 << (sh - 1));
  int64_t q = num >> sh;  // arithmetic shift: floor division
  q = q < 0 ? 0 : q;
  return q > qmax ? qmax : q;
}

__global__ void conv_direct_kernel(ConvArgs a, int chunks, const int32_t *only_if_flag) {
  if (only_if_flag && *only_if_flag == 0) return;
  const int G = a.in.groups;
  const int64_t rows = (int64_t)a.out.n * a.ho * a.wo * G;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= rows * chunks) return;
  const int64_t r = t / chunks;
  const int ci = (int)(t % chunks);
  const int gd = (int)(r % G);                   // destination group
  const int64_t p = r / G;                       // output pixel
  const int ox = (int)(p % a.wo);
  const int oy = (int)((p / a.wo) % a.ho);
  const int n = (int)(p / ((int64_t)a.wo * a.ho));
  const int g = (gd - a.shuffle + G) % G;        // source group
  const int cin = a.in.cpg;
  const int64_t wrow = row_bytes(cin, a.w_bits);
  const int qmax = (1 << a.out.bits) - 1;
  const int j0 = ci * 32;
  const int nc = min(32, a.cout - j0);
  int q[32];
  for (int jj = 0; jj < 32; ++jj) q[jj] = 0;
  for (int jj = 0; jj < nc; ++jj) {
    const int k = j0 + jj;
    int64_t acc = 0;
    for (int ky = 0; ky < a.kh; ++ky) {
      const int iy = oy * a.stride - a.pad + ky;
      if (iy < 0 || iy >= a.in.h) continue;
      for (int kx = 0; kx < a.kw; ++kx) {
        const int ix = ox * a.stride - a.pad + kx;
        if (ix < 0 || ix >= a.in.w) continue;
        const uint8_t *xr = a.in.data + (((int64_t)n * a.in.h + iy) * a.in.w + ix) * a.in.pixel +
                            (int64_t)g * a.in.gstride;
        const uint8_t *wr = a.w + ((((int64_t)g * a.cout + k) * a.kh + ky) * a.kw + kx) * wrow;
        for (int c = 0; c < cin; ++c)
          acc += (int64_t)read_code(xr, c, a.in.bits, a.in.is_signed) * read_code(wr, c, a.w_bits, 1);
      }
    }
    if (a.proj.data) {
      const int iy = oy * a.proj_stride, ix = ox * a.proj_stride;
      const uint8_t *xr = a.proj.data + (((int64_t)n * a.proj.h + iy) * a.proj.w + ix) * a.proj.pixel +
                          (int64_t)gd * a.proj.gstride;
      const int pc = a.proj.cpg;
      const uint8_t *wr = a.proj_w + ((int64_t)gd * a.cout + k) * row_bytes(pc, a.w_bits);
      for (int c = 0; c < pc; ++c)
        acc += (int64_t)read_code(xr, c, a.proj.bits, 0) * read_code(wr, c, a.w_bits, 1);
    }
    const int cs = g * a.cout + k;          // source channel: parameters
    const int cd = gd * a.cout + k;         // destination channel
    if (a.acc_dump) a.acc_dump[p * (int64_t)G * a.cout + cd] = (int32_t)acc;
    int64_t tt = acc + (a.bias ? a.bias[cs] : 0);
    if (a.res.data) {
      const uint8_t *rr = a.res.data + p * a.res.pixel + (int64_t)gd * a.res.gstride;
      tt += (int64_t)a.res_mult[cs] * read_code(rr, k, a.res.bits, 0);
    }
    q[jj] = (int)requant_one(tt, a.mult[cs], a.shift[cs], qmax);
  }
  uint32_t words[8];
  pack_chunk(q, nc, a.out.bits, words);
  const int per_chunk = a.out.bits == 3 ? 3 : store_bits(a.out.bits);
  const int nw = chunk_words_in_row(ci, a.out.bits, a.out.row / 4);
  uint32_t *dst = (uint32_t *)(a.out.data + p * a.out.pixel + (int64_t)gd * a.out.gstride) +
                  (int64_t)ci * per_chunk;
  for (int kk = 0; kk < nw; ++kk) dst[kk] = words[kk];
}

}  // namespace

hipError_t launch_conv_direct(const ConvArgs &a, hipStream_t s, const int32_t *only_if_flag) {
  const int chunks = (a.cout + 31) / 32;
  const int64_t items = (int64_t)a.out.n * a.ho * a.wo * a.in.groups * chunks;
  if (items == 0) return hipSuccess;
  const int64_t grid = (items + 255) / 256;
  hipLaunchKernelGGL(conv_direct_kernel, dim3((unsigned)grid), dim3(256), 0, s, a, chunks, only_if_flag);
  return hipGetLastError();
}

}  // namespace palq
