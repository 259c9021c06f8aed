/*
 * PalQuant CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * Plain, slow, obviously correct reference arithmetic for the parity tests,
 * the smoke check and the CPU baseline leg of the benchmark.  Nothing in the
 * product library links, includes or calls this code, and this code includes
 * nothing from the product library.
 *
 * All tensors here are UNPACKED integer codes (one int32 per code), channels
 * last, with the channel index of a grouped tensor being g * C_per_group + j
 * (the group-major [N, G, C^, H, W] view of the cyclic permutation section,
 * stored NHWC).
 */
#ifndef PALQ_ORACLE_H
#define PALQ_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Grouped convolution with exact int64 accumulation.
 *
 * Follows the matrix-product form of a layer (Preliminaries, Eq. 1) applied
 * independently to each of the G channel groups (Parallel Low-Precision
 * Quantization, Section 4.1: "quantized group convolution with expanded
 * channels").  Out-of-image taps read the code 0.
 *
 *   x   : [n][h][w][groups*cin]              input codes
 *   wt  : [groups][cout][kh][kw][cin]        weight codes
 *   acc : [n][ho][wo][groups*cout]           output, int64
 *   ho = (h + 2*pad - kh) / stride + 1, wo likewise.
 *
 * Returns 0, or -1 on a non-positive size / stride.
 */
int palq_oracle_group_conv(const int32_t *x, int64_t n, int64_t h, int64_t w,
                           int64_t groups, int64_t cin, const int32_t *wt,
                           int64_t cout, int64_t kh, int64_t kw, int64_t stride,
                           int64_t pad, int64_t *acc);

/* Number of threads the conv loop uses (OpenMP team size, 1 without OpenMP). */
int palq_oracle_threads(void);

#ifdef __cplusplus
}
#endif
#endif
