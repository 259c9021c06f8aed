// C ABI of the PalQuant library: context handling, host-side validation of
// every call, and dispatch to the kernels.  Nothing is enqueued before all
// checks pass.
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <new>
#include <string>

#include "palq_internal.h"

using namespace palq;

namespace {

palq_status fail(palq_ctx *ctx, palq_status code, const std::string &msg) {
  if (ctx) ctx->err = msg;
  return code;
}

palq_status device_fail(palq_ctx *ctx, hipError_t e, const char *what) {
  return fail(ctx, PALQ_ERR_DEVICE, std::string(what) + ": " + hipGetErrorString(e));
}

bool valid_bits(int b) { return b == 2 || b == 3 || b == 4 || b == 6 || b == 8; }

int64_t act_elems(const palq_act *a) {
  return (int64_t)a->n * a->h * a->w * a->groups * a->ch_per_group;
}

// Checks a descriptor; `what` names it in the message.
palq_status check_act(palq_ctx *ctx, const palq_act *a, const char *what) {
  if (!a) return fail(ctx, PALQ_ERR_ARG, std::string(what) + ": null descriptor");
  if (a->n < 0 || a->h < 1 || a->w < 1 || a->groups < 1 || a->ch_per_group < 1)
    return fail(ctx, PALQ_ERR_ARG, std::string(what) + ": non-positive size");
  if (!valid_bits(a->bits)) return fail(ctx, PALQ_ERR_ARG, std::string(what) + ": bits not in {2,3,4,6,8}");
  if (a->is_signed != 0 && a->is_signed != 1)
    return fail(ctx, PALQ_ERR_ARG, std::string(what) + ": is_signed must be 0 or 1");
  if (a->layout != PALQ_LAYOUT_PIXEL && a->layout != PALQ_LAYOUT_GROUP)
    return fail(ctx, PALQ_ERR_ARG, std::string(what) + ": layout must be PALQ_LAYOUT_PIXEL or PALQ_LAYOUT_GROUP");
  const int64_t row = row_bytes(a->ch_per_group, a->bits);
  const double bytes = (double)a->n * a->h * a->w * a->groups * (double)row;
  if (bytes > 9.0e18) return fail(ctx, PALQ_ERR_ARG, std::string(what) + ": tensor too large");
  if (a->n > 0 && !a->data) return fail(ctx, PALQ_ERR_ARG, std::string(what) + ": null data");
  if (((uintptr_t)a->data & 15u) != 0)
    return fail(ctx, PALQ_ERR_ARG, std::string(what) + ": data not 16-byte aligned");
  return PALQ_OK;
}

palq_status check_filter(palq_ctx *ctx, const palq_filter *f, const char *what) {
  if (!f) return fail(ctx, PALQ_ERR_ARG, std::string(what) + ": null filter");
  if (f->groups < 1 || f->cout_pg < 1 || f->cin_pg < 1 || f->kh < 1 || f->kw < 1)
    return fail(ctx, PALQ_ERR_ARG, std::string(what) + ": non-positive size");
  if (!valid_bits(f->bits)) return fail(ctx, PALQ_ERR_ARG, std::string(what) + ": bits not in {2,3,4,6,8}");
  if (!f->data) return fail(ctx, PALQ_ERR_ARG, std::string(what) + ": null data");
  if (((uintptr_t)f->data & 15u) != 0)
    return fail(ctx, PALQ_ERR_ARG, std::string(what) + ": data not 16-byte aligned");
  return PALQ_OK;
}

int64_t filter_bytes(const palq_filter *f) {
  return (int64_t)f->groups * f->cout_pg * f->kh * f->kw * row_bytes(f->cin_pg, f->bits);
}

bool overlaps(const void *a, int64_t na, const void *b, int64_t nb) {
  if (!a || !b || na <= 0 || nb <= 0) return false;
  const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
  return a0 < b0 + (uintptr_t)nb && b0 < a0 + (uintptr_t)na;
}

int64_t max_code(int bits, int is_signed) {
  return is_signed ? ((int64_t)1 << (bits - 1)) : (((int64_t)1 << bits) - 1);
}

bool same_shape(const palq_act *a, const palq_act *b) {
  return a->n == b->n && a->h == b->h && a->w == b->w && a->groups == b->groups &&
         a->ch_per_group == b->ch_per_group;
}

}  // namespace

extern "C" {

const char *palq_version(void) { return "palq 0.1 (gfx950)"; }

int64_t palq_row_bytes(int32_t codes, int32_t bits) {
  if (!valid_bits(bits)) return -1;
  return row_bytes(codes, bits);
}

int64_t palq_act_bytes(const palq_act *a) {
  if (!a || a->n < 0 || a->h < 1 || a->w < 1 || a->groups < 1 || a->ch_per_group < 1 ||
      !valid_bits(a->bits))
    return -1;
  return (int64_t)a->n * a->h * a->w * a->groups * row_bytes(a->ch_per_group, a->bits);
}

palq_status palq_create(int32_t device, void *hip_stream, palq_ctx **out) {
  if (!out) return PALQ_ERR_ARG;
  *out = nullptr;
  if (device < -1) return PALQ_ERR_ARG;
  palq_ctx *ctx = new (std::nothrow) palq_ctx();
  if (!ctx) return PALQ_ERR_NOMEM;
  ctx->device = device;
  ctx->stream = (hipStream_t)hip_stream;
  if (const char *e = getenv("PALQ_CONV_FP4")) ctx->conv_fp4 = strcmp(e, "0") != 0;
  if (device >= 0) {
    int count = 0;
    hipError_t e = hipGetDeviceCount(&count);
    if (e != hipSuccess || device >= count) {
      delete ctx;
      return PALQ_ERR_DEVICE;
    }
    e = hipSetDevice(device);
    // the no-alloc call's static buffer: its address on this device, looked
    // up once per device (a failure only disables palq_group_conv_noalloc)
    if (e == hipSuccess) noalloc_scratch_init(device);
    if (e == hipSuccess) e = hipMalloc(&ctx->range_scratch, 2 * sizeof(float));
    if (e == hipSuccess) e = hipEventCreateWithFlags(&ctx->order_event, hipEventDisableTiming);
    if (e != hipSuccess) {
      if (ctx->range_scratch) hipFree(ctx->range_scratch);
      delete ctx;
      return PALQ_ERR_DEVICE;
    }
  }
  *out = ctx;
  return PALQ_OK;
}

void palq_destroy(palq_ctx *ctx) {
  if (!ctx) return;
  if (ctx->device >= 0) {
    hipSetDevice(ctx->device);
    if (ctx->range_scratch) hipFree(ctx->range_scratch);
    if (ctx->conv_scratch) hipFree(ctx->conv_scratch);
    if (ctx->fc_scratch) hipFree(ctx->fc_scratch);
    if (ctx->mod_scratch) hipFree(ctx->mod_scratch);
    if (ctx->order_event) hipEventDestroy(ctx->order_event);
  }
  delete ctx;
}

palq_status palq_set_stream(palq_ctx *ctx, void *hip_stream) {
  if (!ctx) return PALQ_ERR_ARG;
  const hipStream_t ns = (hipStream_t)hip_stream;
  if (ctx->device >= 0 && ns != ctx->stream) {
    // work still queued on the old stream may read the context's scratch
    // (prepacked filters, parameters) that the next call on the new stream
    // overwrites: the new stream waits for everything queued so far
    hipSetDevice(ctx->device);
    hipError_t e = hipEventRecord(ctx->order_event, ctx->stream);
    if (e == hipSuccess) e = hipStreamWaitEvent(ns, ctx->order_event, 0);
    if (e != hipSuccess) return device_fail(ctx, e, "set stream");
  }
  ctx->stream = ns;
  return PALQ_OK;
}

palq_status palq_set_conv_fp4(palq_ctx *ctx, int32_t enable) {
  if (!ctx || (enable != 0 && enable != 1)) return PALQ_ERR_ARG;
  ctx->conv_fp4 = enable;
  return PALQ_OK;
}

palq_status palq_set_conv_bitdecomp(palq_ctx *ctx, int32_t enable) {
  if (!ctx || (enable != 0 && enable != 1)) return PALQ_ERR_ARG;
  ctx->conv_bitdecomp = enable;
  return PALQ_OK;
}

palq_status palq_sync(palq_ctx *ctx) {
  if (!ctx) return PALQ_ERR_ARG;
  if (ctx->device < 0) return PALQ_OK;
  hipSetDevice(ctx->device);
  hipError_t e = hipStreamSynchronize(ctx->stream);
  if (e != hipSuccess) return device_fail(ctx, e, "stream synchronize");
  return PALQ_OK;
}

const char *palq_last_error(const palq_ctx *ctx) { return ctx ? ctx->err.c_str() : "null context"; }

// ------------------------------------------------------------ layout
palq_status palq_pack(palq_ctx *ctx, const void *codes, const palq_act *out) {
  if (!ctx) return PALQ_ERR_ARG;
  palq_status st = check_act(ctx, out, "out");
  if (st) return st;
  if (act_elems(out) > 0 && !codes) return fail(ctx, PALQ_ERR_ARG, "codes: null");
  if (overlaps(codes, act_elems(out), out->data, palq_act_bytes(out)))
    return fail(ctx, PALQ_ERR_ARG, "codes and out overlap");
  if (ctx->device < 0) return PALQ_OK;
  hipSetDevice(ctx->device);
  hipError_t e = launch_pack(codes, view_of(out), ctx->stream);
  return e == hipSuccess ? PALQ_OK : device_fail(ctx, e, "pack");
}

palq_status palq_unpack(palq_ctx *ctx, const palq_act *in, void *codes) {
  if (!ctx) return PALQ_ERR_ARG;
  palq_status st = check_act(ctx, in, "in");
  if (st) return st;
  if (act_elems(in) > 0 && !codes) return fail(ctx, PALQ_ERR_ARG, "codes: null");
  if (overlaps(codes, act_elems(in), in->data, palq_act_bytes(in)))
    return fail(ctx, PALQ_ERR_ARG, "codes and in overlap");
  if (ctx->device < 0) return PALQ_OK;
  hipSetDevice(ctx->device);
  hipError_t e = launch_unpack(view_of(in), codes, ctx->stream);
  return e == hipSuccess ? PALQ_OK : device_fail(ctx, e, "unpack");
}

// ------------------------------------------------------------ quantiser
palq_status palq_quantize(palq_ctx *ctx, const float *x, float l, float u, const palq_act *out,
                          float *range_out) {
  if (!ctx) return PALQ_ERR_ARG;
  palq_status st = check_act(ctx, out, "out");
  if (st) return st;
  const int64_t count = act_elems(out);
  if (count > 0 && !x) return fail(ctx, PALQ_ERR_ARG, "x: null");
  if (((uintptr_t)x & 3u) != 0) return fail(ctx, PALQ_ERR_ARG, "x: not 4-byte aligned");
  const bool calibrate = isnan(l) || isnan(u);
  if (!calibrate) {
    if (!isfinite(l) || !isfinite(u)) return fail(ctx, PALQ_ERR_ARG, "l/u must be finite or NaN");
    if (!(u > l) || !isfinite(u - l)) return fail(ctx, PALQ_ERR_ARG, "need u > l with finite u - l");
  }
  if (overlaps(x, count * 4, out->data, palq_act_bytes(out)))
    return fail(ctx, PALQ_ERR_ARG, "x and out overlap");
  if (range_out && ((uintptr_t)range_out & 3u) != 0)
    return fail(ctx, PALQ_ERR_ARG, "range_out: not 4-byte aligned");
  if (ctx->device < 0) return PALQ_OK;
  hipSetDevice(ctx->device);
  hipError_t e = hipSuccess;
  const ActView ov = view_of(out);
  if (calibrate) {
    e = launch_minmax(x, count, ctx->range_scratch, ctx->stream);
    if (e == hipSuccess && range_out) e = launch_range_out(ctx->range_scratch, range_out, ctx->stream);
    if (e == hipSuccess) e = launch_quantize(x, 0.f, 0.f, ctx->range_scratch, ov, ctx->stream);
  } else {
    if (range_out) {
      const float lu[2] = {l, u};
      e = hipMemcpyAsync(range_out, lu, sizeof(lu), hipMemcpyHostToDevice, ctx->stream);
      if (e == hipSuccess) e = hipStreamSynchronize(ctx->stream);  // lu is on this stack frame
    }
    if (e == hipSuccess) e = launch_quantize(x, l, u, nullptr, ov, ctx->stream);
  }
  return e == hipSuccess ? PALQ_OK : device_fail(ctx, e, "quantize");
}

// ------------------------------------------------------------ shuffle module
// Eq. 9-10 run as the 1x1 layer it equals: the branch is stored one group on
// (Eq. 8 as the write address), the shortcut is the identity residual from
// the module's own input, and the per-group parameters are rotated by one
// group (layer group g takes module group (g + 1) mod G).
palq_status palq_shuffle_module(palq_ctx *ctx, const palq_act *in, const palq_filter *w,
                                const palq_requant *rq, const int32_t *res_mult, const palq_act *out) {
  if (!ctx) return PALQ_ERR_ARG;
  palq_status st;
  if ((st = check_act(ctx, in, "in")) || (st = check_filter(ctx, w, "w"))) return st;
  if (w->kh != 1 || w->kw != 1 || w->cin_pg != w->cout_pg)
    return fail(ctx, PALQ_ERR_ARG, "shuffle module: the filter must be 1x1 with cout_pg == cin_pg");
  if (!rq || !res_mult) return fail(ctx, PALQ_ERR_ARG, "shuffle module: requant and res_mult required");
  palq_residual res{};
  res.identity = in;
  res.res_mult = res_mult;
  {
    palq_ctx vctx;  // every other check is the layer's
    vctx.device = -1;
    st = palq_group_conv(&vctx, in, w, 1, 0, rq, &res, 1, out, nullptr);
    if (st != PALQ_OK) return fail(ctx, st, vctx.err);
  }
  if (ctx->device < 0) return PALQ_OK;
  hipSetDevice(ctx->device);
  const int G = w->groups;
  auto up = [](int64_t b) { return (b + 255) & ~(int64_t)255; };
  const int64_t wb = filter_bytes(w), cb = (int64_t)G * w->cout_pg * 4;
  const int64_t off_m = up(wb), off_s = off_m + up(cb), off_b = off_s + up(cb), off_r = off_b + up(cb);
  const size_t need = (size_t)(off_r + up(cb));
  if (need > ctx->mod_scratch_bytes) {
    if (ctx->mod_scratch) hipFree(ctx->mod_scratch);  // waits for work still reading it
    ctx->mod_scratch = nullptr;
    ctx->mod_scratch_bytes = 0;
    if (hipMalloc(&ctx->mod_scratch, need) != hipSuccess)
      return fail(ctx, PALQ_ERR_NOMEM, "shuffle module: parameter scratch");
    ctx->mod_scratch_bytes = need;
  }
  uint8_t *sc = ctx->mod_scratch;
  hipError_t e = hipSuccess;
  auto rot = [&](int64_t off, const void *src, int64_t bytes) {  // group g <- group g + 1
    const int64_t gb = bytes / G;
    if (e == hipSuccess) e = hipMemcpyAsync(sc + off, (const uint8_t *)src + gb, bytes - gb, hipMemcpyDefault, ctx->stream);
    if (e == hipSuccess) e = hipMemcpyAsync(sc + off + bytes - gb, src, gb, hipMemcpyDefault, ctx->stream);
    return sc + off;
  };
  palq_filter w2 = *w;
  w2.data = rot(0, w->data, wb);
  palq_requant rq2 = *rq;
  rq2.mult = (const int32_t *)rot(off_m, rq->mult, cb);
  rq2.shift = (const int32_t *)rot(off_s, rq->shift, cb);
  rq2.bias = rq->bias ? (const int32_t *)rot(off_b, rq->bias, cb) : nullptr;
  res.res_mult = (const int32_t *)rot(off_r, res_mult, cb);
  if (e != hipSuccess) return device_fail(ctx, e, "shuffle module: parameter copies");
  return palq_group_conv(ctx, in, &w2, 1, 0, &rq2, &res, 1, out, nullptr);
}

// ------------------------------------------------------------ group conv
namespace {
// palq_group_conv (noalloc = false: prepacked filter and constants in the
// context's scratch, grown on demand) and palq_group_conv_noalloc (the
// library's static per-GPU buffer; no allocation, free or synchronisation).
palq_status group_conv_impl(palq_ctx *ctx, const palq_act *in, const palq_filter *w, int32_t stride,
                            int32_t pad, const palq_requant *rq, const palq_residual *res,
                            int32_t shuffle_steps, const palq_act *out, int32_t *acc_dump, bool noalloc) {
  if (!ctx) return PALQ_ERR_ARG;
  palq_status st;
  if ((st = check_act(ctx, in, "in")) || (st = check_filter(ctx, w, "w")) ||
      (st = check_act(ctx, out, "out")))
    return st;
  if (!rq || !rq->mult || !rq->shift) return fail(ctx, PALQ_ERR_ARG, "requant: mult/shift required");
  if (((uintptr_t)rq->mult | (uintptr_t)rq->shift | (uintptr_t)rq->bias) & 15u)
    return fail(ctx, PALQ_ERR_ARG, "requant arrays must be 16-byte aligned");
  if (res && ((uintptr_t)res->res_mult & 15u))
    return fail(ctx, PALQ_ERR_ARG, "res_mult must be 16-byte aligned");
  if (w->groups * (int64_t)w->cout_pg > (1 << 24))
    return fail(ctx, PALQ_ERR_UNSUPPORTED, "more than 2^24 output channels");
  if (!valid_bits(rq->out_bits)) return fail(ctx, PALQ_ERR_ARG, "requant: out_bits not in {2,3,4,6,8}");
  if (stride < 1 || pad < 0) return fail(ctx, PALQ_ERR_ARG, "stride must be >= 1 and pad >= 0");
  if (in->groups != w->groups || in->ch_per_group != w->cin_pg)
    return fail(ctx, PALQ_ERR_ARG, "input groups/channels do not match the filter");
  if (in->is_signed && in->bits != 8)
    return fail(ctx, PALQ_ERR_UNSUPPORTED, "signed input codes must be 8-bit");
  const int64_t ho = ((int64_t)in->h + 2 * pad - w->kh) / stride + 1;
  const int64_t wo = ((int64_t)in->w + 2 * pad - w->kw) / stride + 1;
  if ((int64_t)in->h + 2 * pad < w->kh || (int64_t)in->w + 2 * pad < w->kw || ho < 1 || wo < 1)
    return fail(ctx, PALQ_ERR_ARG, "kernel larger than the padded input");
  if (out->n != in->n || out->h != ho || out->w != wo || out->groups != w->groups ||
      out->ch_per_group != w->cout_pg)
    return fail(ctx, PALQ_ERR_ARG, "output shape does not match the convolution");
  if (out->bits != rq->out_bits || out->is_signed)
    return fail(ctx, PALQ_ERR_ARG, "output must be unsigned codes of requant.out_bits bits");
  const int64_t K = (int64_t)w->kh * w->kw * w->cin_pg;
  // 2-bit inputs: the int8 path carries a factor 16 in its accumulator
  const int64_t lim = (int64_t)1 << (in->bits == 2 ? 26 : 30);
  if (K * max_code(in->bits, in->is_signed) * max_code(w->bits, 1) >= lim)
    return fail(ctx, PALQ_ERR_OVERFLOW, in->bits == 2 ? "accumulator bound K*max|a|*max|w| >= 2^26"
                                                      : "accumulator bound K*max|a|*max|w| >= 2^30");

  const palq_act *rid = res ? res->identity : nullptr;
  const palq_act *pin = res ? res->proj_in : nullptr;
  const palq_filter *pw = res ? res->proj_w : nullptr;
  if (rid && pin) return fail(ctx, PALQ_ERR_ARG, "residual: identity and projection both given");
  if (rid) {
    if ((st = check_act(ctx, rid, "residual.identity"))) return st;
    if (!same_shape(rid, out) || rid->is_signed)
      return fail(ctx, PALQ_ERR_ARG, "identity residual must be unsigned codes of the output's shape");
    if (!res->res_mult) return fail(ctx, PALQ_ERR_ARG, "identity residual needs res_mult");
  }
  if (pin || pw) {
    if (!pin || !pw) return fail(ctx, PALQ_ERR_ARG, "projection needs proj_in and proj_w");
    if ((st = check_act(ctx, pin, "residual.proj_in")) || (st = check_filter(ctx, pw, "residual.proj_w")))
      return st;
    if (pw->kh != 1 || pw->kw != 1 || pw->groups != w->groups || pw->cout_pg != w->cout_pg ||
        pin->groups != pw->groups || pin->ch_per_group != pw->cin_pg)
      return fail(ctx, PALQ_ERR_ARG, "projection filter/input do not match");
    if (pin->is_signed) return fail(ctx, PALQ_ERR_UNSUPPORTED, "projection input must be unsigned codes");
    if (res->proj_stride < 1) return fail(ctx, PALQ_ERR_ARG, "proj_stride must be >= 1");
    if (pin->n != in->n || ((int64_t)pin->h - 1) / res->proj_stride + 1 != ho ||
        ((int64_t)pin->w - 1) / res->proj_stride + 1 != wo)
      return fail(ctx, PALQ_ERR_ARG, "projection output size differs from the convolution's");
    if (K * max_code(in->bits, in->is_signed) * max_code(w->bits, 1) +
            (int64_t)pw->cin_pg * max_code(pin->bits, 0) * max_code(pw->bits, 1) >= lim)
      return fail(ctx, PALQ_ERR_OVERFLOW, "projection accumulator bound over the limit");
  }
  const int64_t ob = palq_act_bytes(out);
  if (overlaps(out->data, ob, in->data, palq_act_bytes(in)) ||
      overlaps(out->data, ob, w->data, filter_bytes(w)) ||
      (rid && overlaps(out->data, ob, rid->data, palq_act_bytes(rid))) ||
      (pin && overlaps(out->data, ob, pin->data, palq_act_bytes(pin))))
    return fail(ctx, PALQ_ERR_ARG, "output overlaps an input");
  const int64_t dump_bytes = (int64_t)out->n * ho * wo * w->groups * w->cout_pg * 4;
  if (acc_dump && (((uintptr_t)acc_dump & 15u) != 0 || overlaps(acc_dump, dump_bytes, out->data, ob)))
    return fail(ctx, PALQ_ERR_ARG, "acc_dump misaligned or overlapping the output");

  ConvArgs a{};
  a.in = view_of(in);
  a.out = view_of(out);
  a.w = (const uint8_t *)w->data;
  a.cout = w->cout_pg; a.kh = w->kh; a.kw = w->kw; a.stride = stride; a.pad = pad;
  a.w_bits = w->bits;
  a.ho = (int32_t)ho; a.wo = (int32_t)wo;
  a.mult = rq->mult; a.shift = rq->shift; a.bias = rq->bias;
  a.shuffle = (int32_t)(((int64_t)shuffle_steps % w->groups + w->groups) % w->groups);
  a.fp4 = ctx->conv_fp4;
  a.bitdecomp = ctx->conv_bitdecomp;
  if (rid) { a.res = view_of(rid); a.res_mult = res->res_mult; }
  if (pin) { a.proj = view_of(pin); a.proj_w = (const uint8_t *)pw->data; a.proj_stride = res->proj_stride; }
  a.acc_dump = acc_dump;
  const bool mfma = conv_mfma_supported(a);
  const ConvPlan plan = mfma ? conv_mfma_plan(a) : ConvPlan{0, 0};
  const size_t wbytes = (plan.w_bytes + 255) & ~(size_t)255;
  const size_t need = wbytes + plan.thr_bytes;
  if (noalloc && need > (size_t)PALQ_NOALLOC_SCRATCH_BYTES)
    return fail(ctx, PALQ_ERR_UNSUPPORTED,
                "no-alloc call: the prepacked filter and requant constants need " + std::to_string(need) +
                    " bytes; the library's static buffer holds " + std::to_string((long long)PALQ_NOALLOC_SCRATCH_BYTES));
  if (ctx->device < 0 || out->n == 0) return PALQ_OK;
  hipSetDevice(ctx->device);
  hipError_t e;
  if (mfma && noalloc) {
    uint8_t *base = noalloc_scratch(ctx->device);
    if (!base) return fail(ctx, PALQ_ERR_DEVICE, "no-alloc call: the static scratch of this device is unavailable");
    uint8_t *wp = base;
    int32_t *thr = (int32_t *)(base + wbytes);
    e = launch_conv_prepare(a, wp, thr, ctx->stream);
    if (e == hipSuccess) e = launch_conv_mfma(a, wp, thr, -1, ctx->stream);
  } else if (mfma) {
    if (need > ctx->conv_scratch_bytes) {
      if (ctx->conv_scratch) hipFree(ctx->conv_scratch);  // waits for work still reading it
      ctx->conv_scratch = nullptr;
      ctx->conv_scratch_bytes = 0;
      if (hipMalloc(&ctx->conv_scratch, need) != hipSuccess)
        return fail(ctx, PALQ_ERR_NOMEM, "conv scratch");
      ctx->conv_scratch_bytes = need;
    }
    uint8_t *wp = ctx->conv_scratch;
    int32_t *thr = (int32_t *)(ctx->conv_scratch + wbytes);
    e = launch_conv_prepare(a, wp, thr, ctx->stream);
    // the epilogue build is not known on the host: both start and the one
    // that applies runs (decided on the device from the requant flag)
    if (e == hipSuccess) e = launch_conv_mfma(a, wp, thr, -1, ctx->stream);
  } else {
    e = launch_conv_direct(a, ctx->stream);
  }
  return e == hipSuccess ? PALQ_OK : device_fail(ctx, e, "group conv");
}
}  // namespace

palq_status palq_group_conv(palq_ctx *ctx, const palq_act *in, const palq_filter *w, int32_t stride,
                            int32_t pad, const palq_requant *rq, const palq_residual *res,
                            int32_t shuffle_steps, const palq_act *out, int32_t *acc_dump) {
  return group_conv_impl(ctx, in, w, stride, pad, rq, res, shuffle_steps, out, acc_dump, false);
}

palq_status palq_group_conv_noalloc(palq_ctx *ctx, const palq_act *in, const palq_filter *w, int32_t stride,
                                    int32_t pad, const palq_requant *rq, const palq_residual *res,
                                    int32_t shuffle_steps, const palq_act *out, int32_t *acc_dump) {
  return group_conv_impl(ctx, in, w, stride, pad, rq, res, shuffle_steps, out, acc_dump, true);
}

// ------------------------------------------------------------ planned layers
namespace {
void *plan_fake(uintptr_t slot) { return (void *)(uintptr_t)(0x100000000ull * (slot + 1)); }

void free_plan(palq_conv_plan *p) {
  if (!p) return;
  if (p->mem && p->ctx && p->ctx->device >= 0) {
    hipSetDevice(p->ctx->device);
    hipFree(p->mem);  // waits for work still reading it
  }
  delete p;
}
}  // namespace

palq_status palq_conv_plan_create(palq_ctx *ctx, const palq_act *in, const palq_filter *w, int32_t stride,
                                  int32_t pad, const palq_requant *rq, const palq_residual *res,
                                  int32_t shuffle_steps, const palq_act *out, palq_conv_plan **plan) {
  if (!ctx || !plan) return PALQ_ERR_ARG;
  *plan = nullptr;
  if (!in || !out) return fail(ctx, PALQ_ERR_ARG, "plan: null descriptor");
  // the layer's checks on stand-in tensor addresses (their data pointers are
  // ignored); the filter, requant and shortcut-scale pointers are the real ones
  palq_act fi = *in, fo = *out, fr{}, fp{};
  fi.data = plan_fake(1);
  fo.data = plan_fake(1000);
  palq_residual fres{};
  const palq_residual *resp = nullptr;
  if (res) {
    fres = *res;
    if (res->identity) { fr = *res->identity; fr.data = plan_fake(2000); fres.identity = &fr; }
    if (res->proj_in) { fp = *res->proj_in; fp.data = plan_fake(3000); fres.proj_in = &fp; }
    resp = &fres;
  }
  {
    palq_ctx vctx;
    vctx.device = -1;
    const palq_status st = palq_group_conv(&vctx, &fi, w, stride, pad, rq, resp, shuffle_steps, &fo, nullptr);
    if (st != PALQ_OK) return fail(ctx, st, "plan: " + vctx.err);
  }
  palq_conv_plan *p = new (std::nothrow) palq_conv_plan();
  if (!p) return fail(ctx, PALQ_ERR_NOMEM, "plan");
  p->ctx = ctx;
  const int G = w->groups;
  const int64_t nch = (int64_t)G * w->cout_pg;
  ConvArgs &a = p->a;
  a.in = view_of(&fi);
  a.out = view_of(&fo);
  a.in.data = a.out.data = nullptr;
  a.cout = w->cout_pg; a.kh = w->kh; a.kw = w->kw; a.stride = stride; a.pad = pad;
  a.w_bits = w->bits;
  a.ho = out->h; a.wo = out->w;
  a.shuffle = (int32_t)(((int64_t)shuffle_steps % G + G) % G);
  a.fp4 = ctx->conv_fp4;
  a.bitdecomp = ctx->conv_bitdecomp;
  p->in_bytes = palq_act_bytes(in);
  p->out_bytes = palq_act_bytes(out);
  p->dump_bytes = (int64_t)out->n * out->h * out->w * nch * 4;
  if (res && res->identity) { a.res = view_of(&fr); a.res.data = nullptr; p->res_kind = 1; p->res_bytes = palq_act_bytes(&fr); }
  if (res && res->proj_in) {
    a.proj = view_of(&fp); a.proj.data = nullptr; a.proj_stride = res->proj_stride;
    p->res_kind = 2; p->res_bytes = palq_act_bytes(&fp);
  }
  if (ctx->device < 0) {  // validate only: nothing to prepare
    *plan = p;
    return PALQ_OK;
  }
  // own copies of the parameters (the caller may free theirs), then the
  // prepacked filter and requant constants
  auto up = [](int64_t b) { return (b + 255) & ~(int64_t)255; };
  const int64_t wb = filter_bytes(w), cb = nch * 4;
  const int64_t pwb = (res && res->proj_w) ? filter_bytes(res->proj_w) : 0;
  int64_t off = 0;
  const int64_t o_w = off; off += up(wb);
  const int64_t o_pw = off; off += up(pwb);
  const int64_t o_m = off; off += up(cb);
  const int64_t o_s = off; off += up(cb);
  const int64_t o_b = off; off += up(cb);
  const int64_t o_r = off; off += up(cb);
  a.in.data = (uint8_t *)plan_fake(1);  // for the kernel choice only: no device access
  a.out.data = (uint8_t *)plan_fake(1000);
  if (a.res.cpg) a.res.data = (uint8_t *)plan_fake(2000);
  if (a.proj.cpg) a.proj.data = (uint8_t *)plan_fake(3000);
  a.proj_w = pwb ? (const uint8_t *)plan_fake(4000) : nullptr;
  p->mfma = conv_mfma_supported(a);
  const ConvPlan cp = p->mfma ? conv_mfma_plan(a) : ConvPlan{0, 0};
  const int64_t o_wp = off; off += up((int64_t)cp.w_bytes);
  const int64_t o_thr = off; off += up((int64_t)cp.thr_bytes);
  hipSetDevice(ctx->device);
  hipError_t e = hipMalloc(&p->mem, (size_t)std::max<int64_t>(off, 256));
  if (e != hipSuccess) { free_plan(p); return fail(ctx, PALQ_ERR_NOMEM, "plan: device memory"); }
  uint8_t *m = (uint8_t *)p->mem;
  auto cp_ = [&](int64_t o, const void *src, int64_t bytes) {
    if (e == hipSuccess && src && bytes > 0) e = hipMemcpyAsync(m + o, src, bytes, hipMemcpyDefault, ctx->stream);
    return src ? m + o : nullptr;
  };
  a.w = cp_(o_w, w->data, wb);
  a.proj_w = pwb ? cp_(o_pw, res->proj_w->data, pwb) : nullptr;
  a.mult = (const int32_t *)cp_(o_m, rq->mult, cb);
  a.shift = (const int32_t *)cp_(o_s, rq->shift, cb);
  a.bias = (const int32_t *)cp_(o_b, rq->bias, cb);
  a.res_mult = (res && res->identity) ? (const int32_t *)cp_(o_r, res->res_mult, cb) : nullptr;
  if (p->mfma) {
    p->wp = m + o_wp;
    p->thr = (int32_t *)(m + o_thr);
    if (e == hipSuccess) e = launch_conv_prepare(a, p->wp, p->thr, ctx->stream);
  }
  if (e == hipSuccess) e = hipStreamSynchronize(ctx->stream);
  if (e != hipSuccess) { free_plan(p); return device_fail(ctx, e, "plan: parameters"); }
  if (p->mfma) {
    p->epi = conv_mfma_epilogue(a, p->thr);
    if (p->epi < 0) { free_plan(p); return fail(ctx, PALQ_ERR_DEVICE, "plan: requant flag"); }
    // a layer too long for the general build's LDS runs its general
    // epilogue on the direct kernel
    if (p->epi == 1 && !conv_mfma_general_fits(a)) p->mfma = false;
    a.f32ep = p->mfma && p->epi == 0 && conv_mfma_f32(a, p->thr);
  }
  a.in.data = a.out.data = a.res.data = a.proj.data = nullptr;
  *plan = p;
  return PALQ_OK;
}

palq_status palq_conv_run(palq_ctx *ctx, const palq_conv_plan *plan, const void *in, const void *res_in, void *out,
                          int32_t *acc_dump) {
  if (!ctx || !plan) return PALQ_ERR_ARG;
  if (plan->ctx != ctx) return fail(ctx, PALQ_ERR_ARG, "plan belongs to another context");
  const bool work = plan->a.out.n > 0;
  if (work && (!in || !out)) return fail(ctx, PALQ_ERR_ARG, "null input or output");
  if (((uintptr_t)in | (uintptr_t)out | (uintptr_t)res_in | (uintptr_t)acc_dump) & 15u)
    return fail(ctx, PALQ_ERR_ARG, "tensors must be 16-byte aligned");
  if (plan->res_kind && work && !res_in) return fail(ctx, PALQ_ERR_ARG, "the plan's shortcut input is missing");
  if (!plan->res_kind && res_in) return fail(ctx, PALQ_ERR_ARG, "the plan has no shortcut input");
  if (overlaps(out, plan->out_bytes, in, plan->in_bytes) || overlaps(out, plan->out_bytes, res_in, plan->res_bytes))
    return fail(ctx, PALQ_ERR_ARG, "output overlaps an input");
  if (acc_dump && (overlaps(acc_dump, plan->dump_bytes, out, plan->out_bytes) ||
                   overlaps(acc_dump, plan->dump_bytes, in, plan->in_bytes)))
    return fail(ctx, PALQ_ERR_ARG, "acc_dump overlaps a tensor");
  if (ctx->device < 0 || !work) return PALQ_OK;
  ConvArgs a = plan->a;
  a.in.data = (uint8_t *)in;
  a.out.data = (uint8_t *)out;
  if (plan->res_kind == 1) a.res.data = (uint8_t *)res_in;
  if (plan->res_kind == 2) a.proj.data = (uint8_t *)res_in;
  a.acc_dump = acc_dump;
  hipSetDevice(ctx->device);
  const hipError_t e = plan->mfma ? launch_conv_mfma(a, plan->wp, plan->thr, plan->epi, ctx->stream)
                                  : launch_conv_direct(a, ctx->stream);
  return e == hipSuccess ? PALQ_OK : device_fail(ctx, e, "conv run");
}

void palq_conv_plan_destroy(palq_conv_plan *plan) { free_plan(plan); }

const char *palq_conv_plan_kernels(const palq_conv_plan *plan) {
  if (!plan) return nullptr;
  if (!plan->ctx || plan->ctx->device < 0) return "";
  return plan->mfma ? conv_kernel_label(plan->a, plan->epi) : "conv_direct_kernel";
}

// ------------------------------------------------------------ shuffle
palq_status palq_cyclic_shuffle(palq_ctx *ctx, const palq_act *in, int32_t steps, const palq_act *out) {
  if (!ctx) return PALQ_ERR_ARG;
  palq_status st;
  if ((st = check_act(ctx, in, "in")) || (st = check_act(ctx, out, "out"))) return st;
  if (!same_shape(in, out) || in->bits != out->bits || in->is_signed != out->is_signed)
    return fail(ctx, PALQ_ERR_ARG, "in and out must have the same shape and bits");
  if (overlaps(in->data, palq_act_bytes(in), out->data, palq_act_bytes(out)))
    return fail(ctx, PALQ_ERR_ARG, "in and out overlap");
  if (ctx->device < 0 || in->n == 0) return PALQ_OK;
  hipSetDevice(ctx->device);
  const int32_t s = (int32_t)(((int64_t)steps % in->groups + in->groups) % in->groups);
  hipError_t e = launch_shuffle(view_of(in), s, view_of(out), ctx->stream);
  return e == hipSuccess ? PALQ_OK : device_fail(ctx, e, "cyclic shuffle");
}

palq_status palq_channel_shuffle(palq_ctx *ctx, const palq_act *in, const palq_act *out) {
  if (!ctx) return PALQ_ERR_ARG;
  palq_status st;
  if ((st = check_act(ctx, in, "in")) || (st = check_act(ctx, out, "out"))) return st;
  if (!same_shape(in, out) || in->bits != out->bits || in->is_signed != out->is_signed)
    return fail(ctx, PALQ_ERR_ARG, "in and out must have the same shape and bits");
  if (overlaps(in->data, palq_act_bytes(in), out->data, palq_act_bytes(out)))
    return fail(ctx, PALQ_ERR_ARG, "in and out overlap");
  if (ctx->device < 0 || in->n == 0) return PALQ_OK;
  hipSetDevice(ctx->device);
  hipError_t e = launch_channel_shuffle(view_of(in), view_of(out), ctx->stream);
  return e == hipSuccess ? PALQ_OK : device_fail(ctx, e, "channel shuffle");
}

// ------------------------------------------------------------ glue
palq_status palq_maxpool(palq_ctx *ctx, const palq_act *in, int32_t k, int32_t stride, int32_t pad,
                         const palq_act *out) {
  if (!ctx) return PALQ_ERR_ARG;
  palq_status st;
  if ((st = check_act(ctx, in, "in")) || (st = check_act(ctx, out, "out"))) return st;
  if (k < 1 || stride < 1 || pad < 0 || pad >= k)
    return fail(ctx, PALQ_ERR_ARG, "need k >= 1, stride >= 1, 0 <= pad < k");
  if (in->is_signed) return fail(ctx, PALQ_ERR_UNSUPPORTED, "max pool takes unsigned codes");
  if ((int64_t)in->h + 2 * pad < k || (int64_t)in->w + 2 * pad < k)
    return fail(ctx, PALQ_ERR_ARG, "window larger than the padded input");
  const int64_t ho = ((int64_t)in->h + 2 * pad - k) / stride + 1;
  const int64_t wo = ((int64_t)in->w + 2 * pad - k) / stride + 1;
  if (out->n != in->n || out->h != ho || out->w != wo || out->groups != in->groups ||
      out->ch_per_group != in->ch_per_group || out->bits != in->bits || out->is_signed)
    return fail(ctx, PALQ_ERR_ARG, "output shape does not match the pool");
  if (overlaps(in->data, palq_act_bytes(in), out->data, palq_act_bytes(out)))
    return fail(ctx, PALQ_ERR_ARG, "in and out overlap");
  if (ctx->device < 0 || in->n == 0) return PALQ_OK;
  hipSetDevice(ctx->device);
  hipError_t e = launch_maxpool(view_of(in), k, stride, pad, view_of(out), ctx->stream);
  return e == hipSuccess ? PALQ_OK : device_fail(ctx, e, "max pool");
}

palq_status palq_avgsum(palq_ctx *ctx, const palq_act *in, int32_t *out) {
  if (!ctx) return PALQ_ERR_ARG;
  palq_status st = check_act(ctx, in, "in");
  if (st) return st;
  if (in->is_signed) return fail(ctx, PALQ_ERR_UNSUPPORTED, "sum takes unsigned codes");
  if (in->n > 0 && (!out || ((uintptr_t)out & 3u)))
    return fail(ctx, PALQ_ERR_ARG, "out: null or misaligned");
  if ((double)in->h * in->w * (double)max_code(in->bits, 0) >= 2147483648.0)
    return fail(ctx, PALQ_ERR_OVERFLOW, "sum may exceed int32");
  if (overlaps(in->data, palq_act_bytes(in), out, (int64_t)in->n * in->groups * in->ch_per_group * 4))
    return fail(ctx, PALQ_ERR_ARG, "in and out overlap");
  if (ctx->device < 0 || in->n == 0) return PALQ_OK;
  hipSetDevice(ctx->device);
  hipError_t e = launch_avgsum(view_of(in), out, ctx->stream);
  return e == hipSuccess ? PALQ_OK : device_fail(ctx, e, "avgsum");
}

palq_status palq_fc(palq_ctx *ctx, const int32_t *x, int32_t n, int32_t cin, const int8_t *w,
                    int32_t cout, int32_t *logits) {
  if (!ctx) return PALQ_ERR_ARG;
  if (n < 0 || cin < 1 || cout < 1) return fail(ctx, PALQ_ERR_ARG, "non-positive size");
  if (n > 0 && (!x || !w || !logits)) return fail(ctx, PALQ_ERR_ARG, "null pointer");
  if (((uintptr_t)x & 3u) || ((uintptr_t)logits & 3u))
    return fail(ctx, PALQ_ERR_ARG, "x/logits not 4-byte aligned");
  if (overlaps(logits, (int64_t)n * cout * 4, x, (int64_t)n * cin * 4) ||
      overlaps(logits, (int64_t)n * cout * 4, w, (int64_t)cout * cin))
    return fail(ctx, PALQ_ERR_ARG, "logits overlap an input");
  if (ctx->device < 0 || n == 0) return PALQ_OK;
  hipSetDevice(ctx->device);
  const size_t need = fc_scratch_bytes(n, cin);
  if (need > ctx->fc_scratch_bytes) {
    if (ctx->fc_scratch) hipFree(ctx->fc_scratch);  // waits for work still reading it
    ctx->fc_scratch = nullptr;
    ctx->fc_scratch_bytes = 0;
    if (hipMalloc(&ctx->fc_scratch, need) != hipSuccess) return fail(ctx, PALQ_ERR_NOMEM, "fc scratch");
    ctx->fc_scratch_bytes = need;
  }
  hipError_t e = launch_fc(x, n, cin, w, cout, logits, need ? ctx->fc_scratch : nullptr, ctx->stream);
  return e == hipSuccess ? PALQ_OK : device_fail(ctx, e, "fc");
}

}  // extern "C"
