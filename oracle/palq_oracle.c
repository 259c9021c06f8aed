/*
 * PalQuant CPU oracle -- TEST INFRASTRUCTURE ONLY (see palq_oracle.h).
 *
 * The grouped convolution written out as its definition: for every output
 * position and every output channel of every group, the sum over the kernel
 * window and that group's input channels of code * weight, in int64.
 * No blocking, no reordering beyond the loop nest of the definition; the
 * outer image-row loop is shared between OpenMP threads, which changes no
 * arithmetic (each output is owned by exactly one thread).
 */
#include "palq_oracle.h"
#ifdef _OPENMP
#include <omp.h>
#endif

int palq_oracle_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

int palq_oracle_group_conv(const int32_t *x, int64_t n, int64_t h, int64_t w,
                           int64_t groups, int64_t cin, const int32_t *wt,
                           int64_t cout, int64_t kh, int64_t kw, int64_t stride,
                           int64_t pad, int64_t *acc) {
  if (n < 0 || h <= 0 || w <= 0 || groups <= 0 || cin <= 0 || cout <= 0 ||
      kh <= 0 || kw <= 0 || stride <= 0 || pad < 0)
    return -1;
  const int64_t ho = (h + 2 * pad - kh) / stride + 1;
  const int64_t wo = (w + 2 * pad - kw) / stride + 1;
  if (ho <= 0 || wo <= 0) return -1;
  const int64_t in_c = groups * cin;    /* channels of one input pixel  */
  const int64_t out_c = groups * cout;  /* channels of one output pixel */

#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int64_t b = 0; b < n; ++b) {
    for (int64_t oy = 0; oy < ho; ++oy) {
      for (int64_t ox = 0; ox < wo; ++ox) {
        for (int64_t g = 0; g < groups; ++g) {
          for (int64_t k = 0; k < cout; ++k) {
            int64_t s = 0;
            for (int64_t ky = 0; ky < kh; ++ky) {
              const int64_t iy = oy * stride - pad + ky;
              if (iy < 0 || iy >= h) continue; /* zero padding */
              for (int64_t kx = 0; kx < kw; ++kx) {
                const int64_t ix = ox * stride - pad + kx;
                if (ix < 0 || ix >= w) continue; /* zero padding */
                const int32_t *xp = x + ((b * h + iy) * w + ix) * in_c + g * cin;
                const int32_t *wp = wt + (((g * cout + k) * kh + ky) * kw + kx) * cin;
                for (int64_t c = 0; c < cin; ++c)
                  s += (int64_t)xp[c] * (int64_t)wp[c];
              }
            }
            acc[((b * ho + oy) * wo + ox) * out_c + g * cout + k] = s;
          }
        }
      }
    }
  }
  return 0;
}
