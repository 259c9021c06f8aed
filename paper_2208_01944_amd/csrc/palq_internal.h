// Internal declarations shared by the library's translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>

#include "palq.h"

namespace palq {

// ----------------------------------------------------------------- layout
// Bytes of a packed row of `codes` codes at `bits` bits (the layout of
// include/palq.h): 4-byte words for b in {2,4,8} (and 6, stored as 8),
// 12-byte chunks of 32 codes for b = 3.
__host__ __device__ inline int64_t row_bytes(int64_t codes, int bits) {
  if (codes <= 0) return -1;
  switch (bits) {
    case 2: case 4: case 8: return 4 * ((codes * bits + 31) / 32);
    case 6: return 4 * ((codes * 8 + 31) / 32);
    case 3: return 12 * ((codes + 31) / 32);
    default: return -1;
  }
}

// True when a row holds exactly its codes (no padding bits), so a pixel's
// rows can be re-grouped without moving data.
__host__ __device__ inline bool row_exact(int64_t codes, int bits) {
  if (bits == 3) return codes % 32 == 0;
  return (codes * (bits == 6 ? 8 : bits)) % 32 == 0;
}

// Device view of an activation tensor.  Row (pixel p, group g) starts at
// data + p * pixel + g * gstride: the pixel layout has pixel = groups * row,
// gstride = row; the group layout pixel = row, gstride = pixels * row.
struct ActView {
  uint8_t *data;
  int32_t n, h, w, groups, cpg, bits, is_signed;
  int64_t row;      // bytes per (pixel, group) row
  int64_t pixel;    // bytes from one pixel's row to the next pixel's (same group)
  int64_t gstride;  // bytes from one group's row to the next group's (same pixel)
  int64_t bytes;    // the whole tensor
};

inline ActView view_of(const palq_act *a) {
  ActView v;
  v.data = (uint8_t *)a->data;
  v.n = a->n; v.h = a->h; v.w = a->w;
  v.groups = a->groups; v.cpg = a->ch_per_group;
  v.bits = a->bits; v.is_signed = a->is_signed;
  v.row = row_bytes(a->ch_per_group, a->bits);
  const int64_t pixels = (int64_t)a->n * a->h * a->w;
  if (a->layout == PALQ_LAYOUT_GROUP) {
    v.pixel = v.row;
    v.gstride = v.row * pixels;
  } else {
    v.pixel = v.row * a->groups;
    v.gstride = v.row;
  }
  v.bytes = v.row * a->groups * pixels;
  return v;
}

// Start of row r of a view, rows counted pixel by pixel (r = p * groups + g).
__host__ __device__ inline uint8_t *row_at(const ActView &v, int64_t r) {
  const int64_t p = r / v.groups, g = r - p * v.groups;
  return v.data + p * v.pixel + g * v.gstride;
}

// ----------------------------------------------------------------- conv
// Everything a conv launch needs, all device pointers.
struct ConvArgs {
  ActView in;            // input codes
  ActView out;           // output codes
  const uint8_t *w;      // packed filter
  int32_t cout, kh, kw, stride, pad, w_bits;
  int32_t ho, wo;
  const int32_t *mult, *shift, *bias;  // bias may be null
  int32_t shuffle;                     // already reduced to [0, G)
  // identity shortcut
  ActView res;           // res.data null when absent
  const int32_t *res_mult;
  // projection shortcut (fused as extra contraction)
  ActView proj;          // proj.data null when absent
  const uint8_t *proj_w;
  int32_t proj_stride;
  int32_t *acc_dump;     // may be null
  int32_t fp4;           // 1: 2-bit layers may run on the FP4 matrix cores (where exact)
  int32_t bitdecomp;     // 1: M-bit layers run as the Eq. 4 bit decomposition on FP4
  int32_t gated;         // set by the launcher: general partner of a tiled launch
  int32_t f32ep;         // 1: the FP4 kernel's exact fp32 requant applies (conv_mfma_f32)
};

// Kernel launchers (return hipError_t of the launch).
// only_if_flag (device, nullable): the kernel does nothing unless *only_if_flag
// is non-zero (the general partner of a tiled launch, see launch_conv_mfma).
hipError_t launch_conv_direct(const ConvArgs &a, hipStream_t s, const int32_t *only_if_flag = nullptr);
// Whether the MFMA kernels take this layer.
bool conv_mfma_supported(const ConvArgs &a);
// Whether the general (persistent, filter-in-LDS) build fits this layer;
// when it does not, a supported layer runs only on the tiled kernel's fast
// epilogue and launch_conv_mfma needs epi == 0.
bool conv_mfma_general_fits(const ConvArgs &a);
// Device scratch the MFMA kernel reads besides the ConvArgs tensors:
// weights in MFMA operand order and, for 2-bit outputs, requant thresholds.
struct ConvPlan {
  size_t w_bytes;
  size_t thr_bytes;
};
ConvPlan conv_mfma_plan(const ConvArgs &a);
// Fills wp (w_bytes) and thr (thr_bytes) for this layer.
hipError_t launch_conv_prepare(const ConvArgs &a, uint8_t *wp, int32_t *thr, hipStream_t s);
// Whether the MFMA path runs faster on a copy of the input with the zero
// border made explicit (launch_pad_pixels, then the same layer with pad 0):
// the 8-bit first layer, whose taps are then fetched without masks.
bool conv_mfma_pads_input(const ConvArgs &a);
// Which epilogue build the layer needs once launch_conv_prepare has run and
// the stream has drained: 0 fast, 1 general, -1 unknown (copy failed).
// Synchronous; for planning only.
int conv_mfma_epilogue(const ConvArgs &a, const int32_t *thr);
// For a layer on the FP4 kernel with the fast epilogue: whether every
// channel's requant is exact in fp32 (written by launch_conv_prepare; reads
// one flag word back, blocking).  Callers keep the answer in ConvArgs::f32ep.
bool conv_mfma_f32(const ConvArgs &a, const int32_t *thr);
// epi: the value above, or -1 when it is not known on the host: both builds
// start and each checks on the device whether it applies (the other returns
// at once); no host synchronisation either way.
hipError_t launch_conv_mfma(const ConvArgs &a, const uint8_t *wp, const int32_t *thr, int epi, hipStream_t s);
// The static per-GPU buffer of palq_group_conv_noalloc (PALQ_NOALLOC_SCRATCH_BYTES):
// noalloc_scratch_init looks its address up on `device` (which must be the
// current device) once per device; noalloc_scratch returns it (nullptr if
// the lookup failed or was not made).
hipError_t noalloc_scratch_init(int device);
uint8_t *noalloc_scratch(int device);
// Kernel family launch_conv_mfma runs for the layer with epi 0 or 1 (static
// string: "conv_tile_kernel[fp4]", "conv_tile_kernel[int8]",
// "conv_tile_kernel[stem]", "conv_grouped_kernel" or "conv_stem_kernel").
const char *conv_kernel_label(const ConvArgs &a, int epi);
// Stem conv fused with the 3x3 / stride 2 / pad 1 max pool of its output
// (written to po only; the stem's own output is not written).  Requires the
// fast epilogue (conv_mfma_epilogue == 0).
bool stem_pool_applies(const ConvArgs &a, const ActView &po, int k, int stride, int pad);
hipError_t launch_stem_pool(const ConvArgs &a, const uint8_t *wp, const int32_t *thr, const ActView &po,
                            hipStream_t s);

hipError_t launch_pack(const void *codes, const ActView &out, hipStream_t s);
hipError_t launch_unpack(const ActView &in, void *codes, hipStream_t s);
hipError_t launch_minmax(const float *x, int64_t count, float *range, hipStream_t s);
hipError_t launch_range_out(const float *enc, float *range_out, hipStream_t s);
hipError_t launch_quantize(const float *x, float l, float u, const float *range, const ActView &out,
                           hipStream_t s);
hipError_t launch_shuffle(const ActView &in, int32_t steps, const ActView &out, hipStream_t s);
hipError_t launch_channel_shuffle(const ActView &in, const ActView &out, hipStream_t s);
const char *channel_shuffle_label(const ActView &in, const ActView &out);
hipError_t launch_maxpool(const ActView &in, int k, int stride, int pad, const ActView &out,
                          hipStream_t s);
hipError_t launch_avgsum(const ActView &in, int32_t *out, hipStream_t s, int8_t *planes = nullptr, int P = 0,
                         int32_t *logits = nullptr, int cout = 0);
// out: in's shape grown by 2 pad pixels in h and w, same pixel bytes.
hipError_t launch_pad_pixels(const ActView &in, int pad, const ActView &out, hipStream_t s);
// Signed 8-bit codes (Eq. 2 with fixed l, u) of an fp32 [n][in_h][in_w][3]
// tensor written into `out`, a 4-byte-pixel tensor of in_h + 2 pad rows and
// in_w + 2 pad columns, zero on the border.
hipError_t launch_quantize_pad(const float *x, float l, float u, int in_h, int in_w, int pad, const ActView &out,
                               hipStream_t s);
// FC: with scratch (fc_scratch_bytes, device) the matrix-core path runs,
// else (or when that returns 0) the vector path.  xmax: a bound on |x| that
// the caller knows (fewer digit planes), or -1.
size_t fc_scratch_bytes(int n, int cin);
hipError_t launch_fc(const int32_t *x, int n, int cin, const int8_t *w, int cout, int32_t *logits,
                     int8_t *scratch, hipStream_t s, int64_t xmax = -1, bool planes_ready = false);
// The matrix-core FC path's conditions; its digit-plane count for |x| <= xmax.
bool fc_mfma_applies(const int32_t *x, int n, int cin, int cout, const int8_t *scratch);
int fc_planes(int64_t xmax);
// Whether the global sum of `in` can also write the FC's digit planes (and
// zero the logits): launch_avgsum with planes != nullptr.
bool avgsum_makes_fc_planes(const ActView &in);

// Names of the kernels the launchers above run for these arguments (static
// strings; the same conditions the launchers test).
const char *quantize_label(const float *x, const ActView &out);
const char *quantize_pad_label(const float *x, int in_w, int pad, const ActView &out);
const char *pad_pixels_label(const ActView &out);
const char *maxpool_label(const ActView &in, const ActView &out);
const char *avgsum_label(const ActView &in, const int32_t *out);
const char *fc_label(const int32_t *x, int n, int cin, int cout, const int8_t *scratch, bool planes_ready);

}  // namespace palq

// The context (opaque to callers).
struct palq_ctx {
  int device = -1;           // -1: validate only
  hipStream_t stream = nullptr;
  std::string err;
  float *range_scratch = nullptr;  // 2 floats for calibration without range_out
  uint8_t *conv_scratch = nullptr; // prepacked weights + thresholds of the last conv call
  size_t conv_scratch_bytes = 0;
  int8_t *fc_scratch = nullptr;    // digit planes of the last FC call
  size_t fc_scratch_bytes = 0;
  int conv_fp4 = 1;                // palq_set_conv_fp4 (initial value: PALQ_CONV_FP4, default 1)
  int conv_bitdecomp = 0;          // palq_set_conv_bitdecomp
  uint8_t *mod_scratch = nullptr;  // rotated parameters of the last shuffle-module call
  size_t mod_scratch_bytes = 0;
  hipEvent_t order_event = nullptr;  // palq_set_stream: the new stream waits for the old one
};

// A planned single layer (palq_conv_plan_create / palq_conv_run).
struct palq_conv_plan {
  palq_ctx *ctx = nullptr;
  palq::ConvArgs a{};        // planned launch (tensor pointers patched per run)
  bool mfma = false;         // matrix-core kernels (else the direct kernel)
  int epi = -1;              // their epilogue build (conv_mfma_epilogue)
  void *mem = nullptr;       // owned device memory: parameters, prepacked filter, constants
  uint8_t *wp = nullptr;
  int32_t *thr = nullptr;
  int64_t in_bytes = 0, out_bytes = 0, res_bytes = 0, dump_bytes = 0;
  int res_kind = 0;          // 0 none, 1 identity codes, 2 projection input
};
