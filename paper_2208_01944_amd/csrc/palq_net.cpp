// Network planner and executor behind palq_net_create / palq_forward.
//
// At create time every layer is validated (through the single-layer entry
// points in validate-only mode), its parameters are copied into one device
// pool owned by the network, tensor shapes are inferred, and activation
// buffers are assigned by liveness (a tensor's buffer is reused once its
// last reader has run).  palq_forward then only patches the input pointer
// and launches the prepared kernels in order on the context's stream.
#include <string.h>

#include <cmath>

#include <algorithm>
#include <new>
#include <string>
#include <vector>

#include "palq_internal.h"

using namespace palq;

namespace {

enum Kind { kCodes = 0, kSums = 1, kLogits = 2 };

struct Tensor {
  bool exists = false;
  int kind = kCodes;
  palq_act d{};          // shape/bits; data filled at plan time
  int64_t bytes = 0;
  int last_use = -1;     // index of the last layer reading it
  int64_t sum_max = -1;  // AVGSUM outputs: bound on every sum
  int buf = -1;          // buffer slot (-1: network input or logits)
};

struct Layer {
  palq_layer spec{};
  // prepared launch arguments (input pointers patched for tensor 0)
  ConvArgs conv{};
  bool use_mfma = false;
  int pad = 0;                   // > 0: the input is first copied with this zero border
  ActView pad_in{};              // the conv's own input (data patched for tensor 0)
  int epi = -1;                  // MFMA epilogue build (conv_mfma_epilogue)
  int32_t *thr = nullptr;        // requant thresholds (2-bit outputs)
  uint8_t *wp = nullptr;         // weights in MFMA operand order
  palq_act in_view{}, out_view{};
  int32_t *sums_out = nullptr;   // AVGSUM
  const int32_t *fc_in = nullptr;
  int8_t *fc_w = nullptr;
  int fc_cin = 0;
  int8_t *fc_scratch = nullptr;  // digit planes of the FC input
  int64_t fc_xmax = -1;          // bound on the FC input (sums of codes)
  // AVGSUM followed by the matrix-core FC: the sum also writes the FC's
  // digit planes (fc_planes_out, P planes) and zeroes the logits
  int8_t *fc_planes_out = nullptr;
  int fc_planes_n = 0, fc_cout = 0;
  bool fc_planes_ready = false;  // FC: skip its own digit pass
  // stem conv whose output only the following max pool reads: one fused
  // launch writes the pooled tensor (pool_out) and the pool layer is skipped
  bool pool_fused = false;
  bool skip = false;
  ActView pool_out{};
};

constexpr int kRing = 64;  // forwards whose layer events can be outstanding

}  // namespace

struct palq_net {
  palq_ctx *ctx = nullptr;
  int flags = 0;
  std::vector<Layer> layers;
  std::vector<Tensor> tensors;
  std::vector<void *> bufs;
  void *pool = nullptr;
  int64_t ops = 0;
  int n = 0, fc_out = 0;
  // timing
  std::vector<hipEvent_t> events;  // kRing * (L + 1)
  std::vector<double> ms;          // per layer
  int pending_begin = 0, pending_end = 0;  // ring indices of unread forwards
  int forwards = 0;
  // palq_forward_image: the input is an 8-bit signed 3-channel image; either
  // every reader of tensor 0 is a conv that copies it with a zero border
  // (img_direct: it quantises straight into that copy) or the image is first
  // quantised into img_codes
  bool img_input = false, img_direct = false;
  void *img_codes = nullptr;
  palq_act input{};
  // PALQ_NET_GRAPH: the replayed graph and the call it was captured for
  bool graph_warm = false;
  hipGraph_t graph = nullptr;
  hipGraphExec_t graph_exec = nullptr;
  hipStream_t cap_stream = nullptr;  // capture only
  const void *g_input = nullptr, *g_img = nullptr;
  int32_t *g_logits = nullptr;
  float g_l = 0.f, g_u = 0.f;
  hipStream_t g_stream = nullptr;
  // palq_net_layer_kernels: per layer, the kernels palq_forward (0) and
  // palq_forward_image (1) launch; img_label: forward_image's own quantiser
  std::vector<std::string> labels[2];
  std::string img_label;
};

namespace {

palq_status net_fail(palq_ctx *ctx, palq_status code, const std::string &msg) {
  if (ctx) ctx->err = msg;
  return code;
}

int64_t act_bytes(const palq_act &a) {
  return (int64_t)a.n * a.h * a.w * a.groups * row_bytes(a.ch_per_group, a.bits);
}

// View tensor t as `groups` rows of cpg codes (same data, same bits).
bool regroup(const palq_act &t, int groups, int cpg, palq_act *out) {
  if ((int64_t)t.groups * t.ch_per_group != (int64_t)groups * cpg) return false;
  // a group-layout tensor keeps each group's rows apart: no other split
  if (t.layout == PALQ_LAYOUT_GROUP && t.groups != groups) return false;
  if (t.groups != groups && !(row_exact(t.ch_per_group, t.bits) && row_exact(cpg, t.bits)))
    return false;
  *out = t;
  out->groups = groups;
  out->ch_per_group = cpg;
  return true;
}

void free_net(palq_net *net) {
  if (!net) return;
  if (net->ctx && net->ctx->device >= 0) hipSetDevice(net->ctx->device);
  for (void *b : net->bufs) if (b) hipFree(b);
  if (net->pool) hipFree(net->pool);
  if (net->img_codes) hipFree(net->img_codes);
  if (net->graph_exec) hipGraphExecDestroy(net->graph_exec);
  if (net->graph) hipGraphDestroy(net->graph);
  if (net->cap_stream) hipStreamDestroy(net->cap_stream);
  for (hipEvent_t e : net->events) if (e) hipEventDestroy(e);
  delete net;
}

// A fake, aligned, non-null device address for validate-only checks.
void *fake_ptr(uintptr_t slot) { return (void *)(uintptr_t)(0x100000000ull * (slot + 1)); }

void accumulate_slot(palq_net *net, int slot) {
  const size_t L = net->layers.size();
  hipEvent_t *ev = &net->events[(size_t)slot * (L + 1)];
  hipEventSynchronize(ev[L]);
  for (size_t i = 0; i < L; ++i) {
    float t = 0.f;
    if (hipEventElapsedTime(&t, ev[i], ev[i + 1]) == hipSuccess) net->ms[i] += t;
  }
  net->forwards += 1;
}

}  // namespace

extern "C" {

palq_status palq_net_create(palq_ctx *ctx, const palq_act *input, const palq_layer *user_layers,
                            int32_t n_layers, int32_t flags, palq_net **out) {
  if (!ctx || !out) return PALQ_ERR_ARG;
  *out = nullptr;
  if (!input || !user_layers || n_layers < 1) return net_fail(ctx, PALQ_ERR_ARG, "empty network");
  // A cyclic shuffle module (Eq. 9-10) is planned as the 1x1 conv layer it
  // equals: branch stored one group on, identity shortcut from its own
  // input, per-group parameters rotated by one group (rotate[i]) when they
  // are copied into the pool.
  std::vector<palq_layer> norm(user_layers, user_layers + n_layers);
  std::vector<char> rotate(n_layers, 0);
  for (int i = 0; i < n_layers; ++i) {
    palq_layer &L = norm[i];
    if (L.op != PALQ_OP_SHUFFLE_MODULE) continue;
    if (L.w.kh != 1 || L.w.kw != 1 || L.w.cin_pg != L.w.cout_pg)
      return net_fail(ctx, PALQ_ERR_ARG, "layer " + std::to_string(i) + ": a shuffle module's filter is 1x1 with cout_pg == cin_pg");
    if (!L.res_mult) return net_fail(ctx, PALQ_ERR_ARG, "layer " + std::to_string(i) + ": res_mult missing");
    L.op = PALQ_OP_CONV;
    L.stride = 1;
    L.pad = 0;
    L.shuffle_steps = 1;
    L.res_src = L.src;
    L.proj_src = -1;
    rotate[i] = 1;
  }
  const palq_layer *layers = norm.data();
  if (flags & ~(PALQ_NET_KEEP_ALL | PALQ_NET_TIMING | PALQ_NET_GRAPH | PALQ_NET_PIXEL_LAYOUT))
    return net_fail(ctx, PALQ_ERR_ARG, "unknown flags");
  if ((flags & PALQ_NET_TIMING) && (flags & PALQ_NET_GRAPH))
    return net_fail(ctx, PALQ_ERR_ARG, "PALQ_NET_GRAPH does not go with PALQ_NET_TIMING");
  if (input->n < 1 || input->h < 1 || input->w < 1 || input->groups < 1 || input->ch_per_group < 1 ||
      row_bytes(input->ch_per_group, input->bits) < 0)
    return net_fail(ctx, PALQ_ERR_ARG, "bad input descriptor");

  palq_ctx vctx;  // validate-only twin of ctx
  vctx.device = -1;
  palq_net *net = new (std::nothrow) palq_net();
  if (!net) return PALQ_ERR_NOMEM;
  net->ctx = ctx;
  net->flags = flags;
  net->layers.resize(n_layers);
  int max_id = 0;
  for (int i = 0; i < n_layers; ++i) max_id = std::max(max_id, layers[i].dst);
  if (max_id < 1 || max_id > 100000) {
    free_net(net);
    return net_fail(ctx, PALQ_ERR_ARG, "tensor ids out of range");
  }
  net->tensors.resize((size_t)max_id + 1);
  Tensor &t0 = net->tensors[0];
  t0.exists = true;
  t0.d = *input;
  t0.d.data = nullptr;
  net->n = input->n;

  // ---- pass 1: shapes and validation
  int64_t pool_bytes = 0;
  auto reserve = [&](int64_t b) { int64_t off = pool_bytes; pool_bytes += (b + 255) & ~(int64_t)255; return off; };
  std::vector<int64_t> off_w(n_layers, -1), off_pw(n_layers, -1), off_mult(n_layers, -1),
      off_shift(n_layers, -1), off_bias(n_layers, -1), off_rm(n_layers, -1), off_fc(n_layers, -1),
      off_thr(n_layers, -1);
  std::string err;
  palq_status st = PALQ_OK;
  for (int i = 0; i < n_layers && st == PALQ_OK; ++i) {
    const palq_layer &L = layers[i];
    Layer &NL = net->layers[i];
    NL.spec = L;
    char where[64];
    snprintf(where, sizeof where, "layer %d: ", i);
    auto bad = [&](palq_status code, const std::string &m) { st = code; err = where + m; };
    if (L.dst <= 0 || L.dst > max_id || net->tensors[L.dst].exists) { bad(PALQ_ERR_ARG, "dst id reused or invalid"); break; }
    if (L.src < 0 || L.src >= L.dst || !net->tensors[L.src].exists) { bad(PALQ_ERR_ARG, "src is not an earlier tensor"); break; }
    Tensor &src = net->tensors[L.src];
    src.last_use = i;
    Tensor &dst = net->tensors[L.dst];
    if (L.op == PALQ_OP_CONV) {
      if (src.kind != kCodes) { bad(PALQ_ERR_ARG, "conv input must be codes"); break; }
      palq_act in_v;
      if (!regroup(src.d, L.w.groups, L.w.cin_pg, &in_v)) { bad(PALQ_ERR_ARG, "input cannot be viewed with the filter's groups"); break; }
      if (L.stride < 1 || L.pad < 0 || L.w.kh < 1 || L.w.kw < 1 ||
          (int64_t)in_v.h + 2 * L.pad < L.w.kh || (int64_t)in_v.w + 2 * L.pad < L.w.kw) {
        bad(PALQ_ERR_ARG, "bad conv geometry"); break;
      }
      palq_act o{};
      o.n = in_v.n; o.groups = L.w.groups; o.ch_per_group = L.w.cout_pg;
      o.h = (in_v.h + 2 * L.pad - L.w.kh) / L.stride + 1;
      o.w = (in_v.w + 2 * L.pad - L.w.kw) / L.stride + 1;
      o.bits = L.out_bits; o.is_signed = 0;
      // validate with the single-layer checks on fake addresses
      palq_act fi = in_v, fo = o, fr{}, fp{};
      fi.data = fake_ptr(1); fo.data = fake_ptr(1000);
      palq_filter fw = L.w; fw.data = fake_ptr(2000);
      palq_filter fpw = L.proj_w; fpw.data = fake_ptr(3000);
      palq_requant rq{(const int32_t *)fake_ptr(4000), (const int32_t *)fake_ptr(4001),
                      L.bias ? (const int32_t *)fake_ptr(4002) : nullptr, L.out_bits};
      palq_residual res{};
      if (L.res_src >= 0 && L.proj_src >= 0) { bad(PALQ_ERR_ARG, "both identity and projection shortcuts"); break; }
      if (L.res_src >= 0) {
        if (L.res_src >= L.dst || !net->tensors[L.res_src].exists || net->tensors[L.res_src].kind != kCodes) { bad(PALQ_ERR_ARG, "res_src is not an earlier code tensor"); break; }
        if (!regroup(net->tensors[L.res_src].d, o.groups, o.ch_per_group, &fr)) { bad(PALQ_ERR_ARG, "residual cannot be viewed with the output's groups"); break; }
        if (!L.res_mult) { bad(PALQ_ERR_ARG, "res_mult missing"); break; }
        net->tensors[L.res_src].last_use = i;
        fr.data = fake_ptr(5000);
        res.identity = &fr;
        res.res_mult = (const int32_t *)fake_ptr(5001);
      }
      if (L.proj_src >= 0) {
        if (L.proj_src >= L.dst || !net->tensors[L.proj_src].exists || net->tensors[L.proj_src].kind != kCodes) { bad(PALQ_ERR_ARG, "proj_src is not an earlier code tensor"); break; }
        if (!regroup(net->tensors[L.proj_src].d, L.proj_w.groups, L.proj_w.cin_pg, &fp)) { bad(PALQ_ERR_ARG, "projection input cannot be viewed with its filter's groups"); break; }
        net->tensors[L.proj_src].last_use = i;
        fp.data = fake_ptr(6000);
        res.proj_in = &fp;
        res.proj_w = &fpw;
        res.proj_stride = L.proj_stride;
      }
      if (!L.w.data || !L.mult || !L.shift || (L.proj_src >= 0 && !L.proj_w.data)) { bad(PALQ_ERR_ARG, "null parameter pointer"); break; }
      palq_status s2 = palq_group_conv(&vctx, &fi, &fw, L.stride, L.pad, &rq,
                                       (res.identity || res.proj_in) ? &res : nullptr,
                                       L.shuffle_steps, &fo, nullptr);
      if (s2 != PALQ_OK) { bad(s2, vctx.err); break; }
      dst.exists = true; dst.kind = kCodes; dst.d = o;
      const int64_t nch = (int64_t)L.w.groups * L.w.cout_pg;
      off_w[i] = reserve((int64_t)L.w.groups * L.w.cout_pg * L.w.kh * L.w.kw * row_bytes(L.w.cin_pg, L.w.bits));
      off_mult[i] = reserve(nch * 4);
      off_shift[i] = reserve(nch * 4);
      if (L.bias) off_bias[i] = reserve(nch * 4);
      if (L.res_src >= 0) off_rm[i] = reserve(nch * 4);

      if (L.proj_src >= 0)
        off_pw[i] = reserve((int64_t)L.proj_w.groups * L.proj_w.cout_pg * row_bytes(L.proj_w.cin_pg, L.proj_w.bits));
      const int64_t mac = (int64_t)o.n * o.h * o.w * nch *
                          ((int64_t)L.w.kh * L.w.kw * L.w.cin_pg + (L.proj_src >= 0 ? L.proj_w.cin_pg : 0));
      net->ops += 2 * mac;
      NL.in_view = in_v;
      NL.out_view = o;
    } else if (L.op == PALQ_OP_CHANNEL_SHUFFLE) {
      if (src.kind != kCodes) { bad(PALQ_ERR_ARG, "channel shuffle input must be codes"); break; }
      dst.exists = true; dst.kind = kCodes; dst.d = src.d;
      NL.in_view = src.d; NL.out_view = src.d;
    } else if (L.op == PALQ_OP_MAXPOOL) {
      if (src.kind != kCodes || src.d.is_signed) { bad(PALQ_ERR_ARG, "max pool input must be unsigned codes"); break; }
      if (L.pool_k < 1 || L.pool_stride < 1 || L.pool_pad < 0 || L.pool_pad >= L.pool_k ||
          (int64_t)src.d.h + 2 * L.pool_pad < L.pool_k || (int64_t)src.d.w + 2 * L.pool_pad < L.pool_k) {
        bad(PALQ_ERR_ARG, "bad pool geometry"); break;
      }
      palq_act o = src.d;
      o.h = (src.d.h + 2 * L.pool_pad - L.pool_k) / L.pool_stride + 1;
      o.w = (src.d.w + 2 * L.pool_pad - L.pool_k) / L.pool_stride + 1;
      dst.exists = true; dst.kind = kCodes; dst.d = o;
      NL.in_view = src.d; NL.out_view = o;
    } else if (L.op == PALQ_OP_AVGSUM) {
      if (src.kind != kCodes || src.d.is_signed) { bad(PALQ_ERR_ARG, "sum input must be unsigned codes"); break; }
      palq_act o{};
      o.n = src.d.n; o.h = 1; o.w = 1; o.groups = 1; o.ch_per_group = src.d.groups * src.d.ch_per_group;
      o.bits = 32; o.is_signed = 1;
      dst.exists = true; dst.kind = kSums; dst.d = o;
      dst.sum_max = (((int64_t)1 << src.d.bits) - 1) * src.d.h * src.d.w;
      NL.in_view = src.d; NL.out_view = o;
    } else if (L.op == PALQ_OP_FC) {
      if (src.kind != kSums) { bad(PALQ_ERR_ARG, "FC input must be an AVGSUM output"); break; }
      if (L.fc_out < 1 || !L.fc_w) { bad(PALQ_ERR_ARG, "FC needs fc_w and fc_out >= 1"); break; }
      if (i != n_layers - 1) { bad(PALQ_ERR_ARG, "FC must be the last layer"); break; }
      palq_act o{};
      o.n = src.d.n; o.h = 1; o.w = 1; o.groups = 1; o.ch_per_group = L.fc_out; o.bits = 32; o.is_signed = 1;
      dst.exists = true; dst.kind = kLogits; dst.d = o;
      NL.fc_cin = src.d.ch_per_group;
      NL.fc_xmax = src.sum_max;
      off_fc[i] = reserve((int64_t)L.fc_out * NL.fc_cin);
      net->ops += 2 * (int64_t)o.n * L.fc_out * NL.fc_cin;
      net->fc_out = L.fc_out;
      NL.in_view = src.d; NL.out_view = o;
    } else {
      bad(PALQ_ERR_ARG, "unknown op");
    }
  }
  if (st == PALQ_OK && layers[n_layers - 1].op != PALQ_OP_FC) {
    st = PALQ_ERR_ARG;
    err = "the last layer must be PALQ_OP_FC";
  }
  if (st != PALQ_OK) {
    free_net(net);
    return net_fail(ctx, st, err);
  }
  // ---- tensor layouts: a conv, channel shuffle or max pool output of
  // several groups whose every reader takes it with those groups is stored
  // group by group (PALQ_LAYOUT_GROUP), so that a tile of one group's
  // pixels is one contiguous run for the conv operand fetches, shortcut
  // reads and stores
  if (!(flags & PALQ_NET_PIXEL_LAYOUT)) {
    std::vector<char> grouped_out(net->tensors.size(), 0), split(net->tensors.size(), 0);
    for (int i = 0; i < n_layers; ++i) {
      const palq_layer &L = layers[i];
      if (L.op == PALQ_OP_CHANNEL_SHUFFLE || L.op == PALQ_OP_MAXPOOL) grouped_out[L.dst] = 1;
      if (L.op != PALQ_OP_CONV) continue;
      grouped_out[L.dst] = 1;
      if (L.w.groups != net->tensors[L.src].d.groups) split[L.src] = 1;
      if (L.res_src >= 0 && L.w.groups != net->tensors[L.res_src].d.groups) split[L.res_src] = 1;
      if (L.proj_src >= 0 && L.proj_w.groups != net->tensors[L.proj_src].d.groups) split[L.proj_src] = 1;
    }
    for (size_t t = 1; t < net->tensors.size(); ++t) {
      Tensor &T = net->tensors[t];
      if (T.exists && T.kind == kCodes && grouped_out[t] && !split[t] && T.d.groups > 1) T.d.layout = PALQ_LAYOUT_GROUP;
    }
    for (int i = 0; i < n_layers; ++i) {
      const palq_layer &L = layers[i];
      Layer &NL = net->layers[i];
      if (L.op != PALQ_OP_CONV) continue;
      NL.in_view.layout = net->tensors[L.src].d.layout;
      NL.out_view.layout = net->tensors[L.dst].d.layout;
    }
  }
  net->input = *input;  // palq_forward_image's input format
  net->img_input = input->bits == 8 && input->is_signed && input->groups == 1 && input->ch_per_group == 3;
  if (ctx->device < 0) {  // validate-only context: nothing to allocate
    *out = net;
    return PALQ_OK;
  }

  // ---- pass 2: device memory
  hipSetDevice(ctx->device);
  hipError_t e = hipMalloc(&net->pool, pool_bytes > 0 ? pool_bytes : 256);
  if (e != hipSuccess) { free_net(net); return net_fail(ctx, PALQ_ERR_NOMEM, "parameter pool"); }
  uint8_t *pool = (uint8_t *)net->pool;
  for (int i = 0; i < n_layers && e == hipSuccess; ++i) {
    const palq_layer &L = layers[i];
    Layer &NL = net->layers[i];
    // group-major arrays; rotated: group g of the copy is group (g + 1) mod G
    // of the source (a shuffle module, see above)
    const int rot_groups = rotate[i] ? L.w.groups : 1;
    auto cp = [&](int64_t off, const void *src, int64_t bytes) {
      if (e == hipSuccess && bytes > 0) {
        const int64_t gb = bytes / rot_groups;
        const uint8_t *s8 = (const uint8_t *)src;
        if (rot_groups > 1) {
          e = hipMemcpyAsync(pool + off, s8 + gb, bytes - gb, hipMemcpyDefault, ctx->stream);
          if (e == hipSuccess) e = hipMemcpyAsync(pool + off + bytes - gb, s8, gb, hipMemcpyDefault, ctx->stream);
        } else {
          e = hipMemcpyAsync(pool + off, src, bytes, hipMemcpyDefault, ctx->stream);
        }
      }
      return pool + off;
    };
    if (L.op == PALQ_OP_CONV) {
      const int64_t nch = (int64_t)L.w.groups * L.w.cout_pg;
      ConvArgs &a = NL.conv;
      a.w = cp(off_w[i], L.w.data, (int64_t)L.w.groups * L.w.cout_pg * L.w.kh * L.w.kw * row_bytes(L.w.cin_pg, L.w.bits));
      a.mult = (const int32_t *)cp(off_mult[i], L.mult, nch * 4);
      a.shift = (const int32_t *)cp(off_shift[i], L.shift, nch * 4);
      a.bias = L.bias ? (const int32_t *)cp(off_bias[i], L.bias, nch * 4) : nullptr;
      a.res_mult = L.res_src >= 0 ? (const int32_t *)cp(off_rm[i], L.res_mult, nch * 4) : nullptr;
      a.proj_w = L.proj_src >= 0 ? cp(off_pw[i], L.proj_w.data, (int64_t)L.proj_w.groups * L.proj_w.cout_pg * row_bytes(L.proj_w.cin_pg, L.proj_w.bits)) : nullptr;
      a.cout = L.w.cout_pg; a.kh = L.w.kh; a.kw = L.w.kw; a.stride = L.stride; a.pad = L.pad;
      a.w_bits = L.w.bits;
      a.fp4 = ctx->conv_fp4;
      a.bitdecomp = ctx->conv_bitdecomp;
      a.ho = NL.out_view.h; a.wo = NL.out_view.w;
      a.shuffle = (int32_t)(((int64_t)L.shuffle_steps % L.w.groups + L.w.groups) % L.w.groups);
      a.proj_stride = L.proj_stride;
    } else if (L.op == PALQ_OP_FC) {
      NL.fc_w = (int8_t *)cp(off_fc[i], L.fc_w, (int64_t)L.fc_out * NL.fc_cin);
    }
  }
  if (e == hipSuccess) e = hipStreamSynchronize(ctx->stream);
  if (e != hipSuccess) { free_net(net); return net_fail(ctx, PALQ_ERR_DEVICE, "copying parameters"); }

  // ---- buffers by liveness
  std::vector<int64_t> buf_size;
  std::vector<int> buf_free_after;  // layer index after which the slot is free
  for (int i = 0; i < n_layers; ++i) {
    Tensor &t = net->tensors[layers[i].dst];
    if (t.kind == kLogits) continue;
    t.bytes = t.kind == kSums ? (int64_t)t.d.n * t.d.ch_per_group * 4 : act_bytes(t.d);
    int pick = -1;
    if (!(flags & PALQ_NET_KEEP_ALL)) {
      for (size_t b = 0; b < buf_size.size(); ++b)
        if (buf_free_after[b] < i && (pick < 0 || buf_size[b] < buf_size[pick]) && buf_size[b] >= t.bytes) pick = (int)b;
      if (pick < 0)  // grow the largest free slot instead of adding one
        for (size_t b = 0; b < buf_size.size(); ++b)
          if (buf_free_after[b] < i && (pick < 0 || buf_size[b] > buf_size[pick])) pick = (int)b;
    }
    if (pick < 0) {
      buf_size.push_back(0);
      buf_free_after.push_back(0);
      pick = (int)buf_size.size() - 1;
    }
    buf_size[pick] = std::max(buf_size[pick], t.bytes);
    // a tensor nobody reads is still kept until the end (inspection)
    buf_free_after[pick] = t.last_use < 0 ? n_layers : t.last_use;
    t.buf = pick;
  }
  net->bufs.assign(buf_size.size(), nullptr);
  for (size_t b = 0; b < buf_size.size(); ++b) {
    if (hipMalloc(&net->bufs[b], buf_size[b] > 0 ? buf_size[b] : 256) != hipSuccess) {
      free_net(net);
      return net_fail(ctx, PALQ_ERR_NOMEM, "activation buffers");
    }
  }
  for (auto &t : net->tensors)
    if (t.exists && t.buf >= 0) t.d.data = net->bufs[t.buf];

  // ---- patch tensor pointers into the prepared launches
  for (int i = 0; i < n_layers; ++i) {
    const palq_layer &L = layers[i];
    Layer &NL = net->layers[i];
    if (L.op == PALQ_OP_CONV) {
      ConvArgs &a = NL.conv;
      palq_act iv = NL.in_view; iv.data = net->tensors[L.src].d.data;
      palq_act ov = NL.out_view; ov.data = net->tensors[L.dst].d.data;
      a.in = view_of(&iv);
      a.out = view_of(&ov);
      if (L.res_src >= 0) {
        palq_act rv;
        regroup(net->tensors[L.res_src].d, ov.groups, ov.ch_per_group, &rv);
        a.res = view_of(&rv);
      }
      if (L.proj_src >= 0) {
        palq_act pv;
        regroup(net->tensors[L.proj_src].d, L.proj_w.groups, L.proj_w.cin_pg, &pv);
        a.proj = view_of(&pv);
      }
      NL.use_mfma = conv_mfma_supported(a);
      if (NL.use_mfma && conv_mfma_pads_input(a)) {
        palq_act pv = iv;
        pv.h += 2 * a.pad;
        pv.w += 2 * a.pad;
        void *mem = nullptr;
        if (hipMalloc(&mem, (size_t)act_bytes(pv) + 256) != hipSuccess) {
          free_net(net);
          return net_fail(ctx, PALQ_ERR_NOMEM, "padded input");
        }
        net->bufs.push_back(mem);
        pv.data = mem;
        NL.pad = a.pad;
        NL.pad_in = a.in;
        a.in = view_of(&pv);
        a.pad = 0;
      }
      if (NL.use_mfma) {
        const ConvPlan plan = conv_mfma_plan(a);
        void *mem = nullptr;
        if (hipMalloc(&mem, ((plan.w_bytes + 255) & ~(size_t)255) + plan.thr_bytes + 256) != hipSuccess) {
          free_net(net);
          return net_fail(ctx, PALQ_ERR_NOMEM, "prepacked weights");
        }
        net->bufs.push_back(mem);  // freed with the activation buffers
        NL.wp = (uint8_t *)mem;
        NL.thr = (int32_t *)((uint8_t *)mem + ((plan.w_bytes + 255) & ~(size_t)255));
        if (launch_conv_prepare(a, NL.wp, NL.thr, ctx->stream) != hipSuccess) {
          free_net(net);
          return net_fail(ctx, PALQ_ERR_DEVICE, "weight prepack");
        }
      }
    } else if (L.op == PALQ_OP_AVGSUM) {
      NL.sums_out = (int32_t *)net->tensors[L.dst].d.data;
    } else if (L.op == PALQ_OP_FC) {
      NL.fc_in = (const int32_t *)net->tensors[L.src].d.data;
      const size_t need = fc_scratch_bytes(net->n, NL.fc_cin);
      if (need) {
        void *mem = nullptr;
        if (hipMalloc(&mem, need) != hipSuccess) {
          free_net(net);
          return net_fail(ctx, PALQ_ERR_NOMEM, "fc scratch");
        }
        net->bufs.push_back(mem);
        NL.fc_scratch = (int8_t *)mem;
      }
    }
  }

  // global sum + matrix-core FC: the sum writes the FC's digit planes
  for (int i = 0; i + 1 < n_layers; ++i) {
    Layer &A = net->layers[i], &F = net->layers[i + 1];
    if (layers[i].op != PALQ_OP_AVGSUM || layers[i + 1].op != PALQ_OP_FC || layers[i + 1].src != layers[i].dst)
      continue;
    const palq_act &src = net->tensors[layers[i].src].d;
    if (layers[i].src == 0 || !avgsum_makes_fc_planes(view_of(&src)) ||
        !fc_mfma_applies(F.fc_in, net->n, F.fc_cin, layers[i + 1].fc_out, F.fc_scratch))
      continue;
    A.fc_planes_out = F.fc_scratch;
    A.fc_planes_n = fc_planes(F.fc_xmax);
    A.fc_cout = layers[i + 1].fc_out;
    F.fc_planes_ready = true;
  }
  if (hipStreamSynchronize(ctx->stream) != hipSuccess) {
    free_net(net);
    return net_fail(ctx, PALQ_ERR_DEVICE, "requant thresholds");
  }
  // the requant constants are final: fix each MFMA layer's epilogue build
  for (Layer &NL : net->layers)
    if (NL.spec.op == PALQ_OP_CONV && NL.use_mfma) {
      NL.epi = conv_mfma_epilogue(NL.conv, NL.thr);
      // a layer too long for the general build's LDS runs its general
      // epilogue on the direct kernel
      if (NL.epi != 0 && !conv_mfma_general_fits(NL.conv)) NL.use_mfma = false;
      NL.conv.f32ep = NL.use_mfma && NL.epi == 0 && conv_mfma_f32(NL.conv, NL.thr);
    }
  // fuse the stem with a max pool that is its output's only reader
  if (!(flags & PALQ_NET_KEEP_ALL))
    for (int i = 0; i + 1 < n_layers; ++i) {
      Layer &NL = net->layers[i];
      const palq_layer &P = layers[i + 1];
      if (layers[i].op != PALQ_OP_CONV || !NL.use_mfma || NL.epi != 0 || P.op != PALQ_OP_MAXPOOL ||
          P.src != layers[i].dst || net->tensors[layers[i].dst].last_use != i + 1)
        continue;
      const ActView po = view_of(&net->tensors[P.dst].d);
      if (!stem_pool_applies(NL.conv, po, P.pool_k, P.pool_stride, P.pool_pad)) continue;
      NL.pool_fused = true;
      NL.pool_out = po;
      net->layers[i + 1].skip = true;
    }
  // palq_forward_image: quantise straight into the zero-border copies when
  // they are the only readers of tensor 0, else into a buffer of its own
  if (net->img_input) {
    bool direct = true;
    for (int i = 0; i < n_layers; ++i) {
      const palq_layer &L = layers[i];
      const bool conv = L.op == PALQ_OP_CONV;
      const bool reads0 = L.src == 0 || (conv && (L.res_src == 0 || L.proj_src == 0));
      if (reads0 && !(conv && L.src == 0 && net->layers[i].pad > 0 && L.res_src != 0 && L.proj_src != 0))
        direct = false;
    }
    net->img_direct = direct;
    if (!direct) {
      if (hipMalloc(&net->img_codes, (size_t)act_bytes(*input) + 256) != hipSuccess) {
        free_net(net);
        return net_fail(ctx, PALQ_ERR_NOMEM, "image codes");
      }
      net->input.data = net->img_codes;
    }
  }
  // the kernels each layer launches (the launchers' own selection rules)
  for (int v = 0; v < 2; ++v) net->labels[v].assign(n_layers, std::string());
  for (int i = 0; i < n_layers; ++i) {
    const palq_layer &L = layers[i];
    const Layer &NL = net->layers[i];
    if (NL.skip) continue;
    std::string k;
    if (L.op == PALQ_OP_CONV) {
      k = NL.pool_fused ? "stem_pool_kernel" : NL.use_mfma ? conv_kernel_label(NL.conv, NL.epi) : "conv_direct_kernel";
    } else if (L.op == PALQ_OP_CHANNEL_SHUFFLE) {
      k = channel_shuffle_label(view_of(&net->tensors[L.src].d), view_of(&net->tensors[L.dst].d));
    } else if (L.op == PALQ_OP_MAXPOOL) {
      k = maxpool_label(view_of(&net->tensors[L.src].d), view_of(&net->tensors[L.dst].d));
    } else if (L.op == PALQ_OP_AVGSUM) {
      k = avgsum_label(view_of(&net->tensors[L.src].d), NL.sums_out);
    } else if (L.op == PALQ_OP_FC) {
      k = fc_label(NL.fc_in, net->n, NL.fc_cin, L.fc_out, NL.fc_scratch, NL.fc_planes_ready);
    }
    net->labels[0][i] = net->labels[1][i] = k;
    if (L.op == PALQ_OP_CONV && NL.pad > 0) {
      net->labels[0][i] = std::string(pad_pixels_label(NL.conv.in)) + " + " + k;
      net->labels[1][i] = (net->img_direct && L.src == 0)
                              ? std::string(quantize_pad_label((const float *)fake_ptr(0), NL.pad_in.w, NL.pad, NL.conv.in)) + " + " + k
                              : net->labels[0][i];
    }
  }
  if (net->img_input && !net->img_direct) net->img_label = quantize_label((const float *)fake_ptr(0), view_of(&net->input));
  if (flags & PALQ_NET_TIMING) {
    net->events.assign((size_t)kRing * (n_layers + 1), nullptr);
    for (auto &ev : net->events)
      if (hipEventCreate(&ev) != hipSuccess) { free_net(net); return net_fail(ctx, PALQ_ERR_DEVICE, "events"); }
    net->ms.assign(n_layers, 0.0);
  }
  *out = net;
  return PALQ_OK;
}

void palq_net_destroy(palq_net *net) { free_net(net); }

int64_t palq_net_ops(const palq_net *net) { return net ? net->ops : -1; }

namespace {
// img != nullptr: the layers that read tensor 0 through a zero-border copy
// quantise img (fp32, Eq. 2 with l, u) into that copy instead (img_direct).
palq_status forward_impl(palq_ctx *ctx, palq_net *net, const void *input, int32_t *logits, const float *img,
                         float l, float u, hipStream_t s) {
  const size_t L = net->layers.size();
  hipEvent_t *ev = nullptr;
  if (net->flags & PALQ_NET_TIMING) {
    if (net->pending_end - net->pending_begin >= kRing) {
      accumulate_slot(net, net->pending_begin % kRing);
      net->pending_begin += 1;
    }
    ev = &net->events[(size_t)(net->pending_end % kRing) * (L + 1)];
    net->pending_end += 1;
    hipEventRecord(ev[0], s);
  }
  hipError_t e = hipSuccess;
  for (size_t i = 0; i < L && e == hipSuccess; ++i) {
    Layer &NL = net->layers[i];
    const palq_layer &sp = NL.spec;
    if (NL.skip) {
      if (ev) hipEventRecord(ev[i + 1], s);
      continue;
    }
    switch (sp.op) {
      case PALQ_OP_CONV: {
        ConvArgs a = NL.conv;
        if (NL.pad > 0 && img && sp.src == 0) {
          e = launch_quantize_pad(img, l, u, NL.pad_in.h, NL.pad_in.w, NL.pad, a.in, s);
          if (e != hipSuccess) break;
        } else if (NL.pad > 0) {
          ActView src = NL.pad_in;
          if (sp.src == 0) src.data = (uint8_t *)input;
          e = launch_pad_pixels(src, NL.pad, a.in, s);
          if (e != hipSuccess) break;
        } else if (sp.src == 0) {
          a.in.data = (uint8_t *)input;
        }
        if (sp.res_src == 0) a.res.data = (uint8_t *)input;
        if (sp.proj_src == 0) a.proj.data = (uint8_t *)input;
        if (NL.pool_fused) e = launch_stem_pool(a, NL.wp, NL.thr, NL.pool_out, s);
        else e = NL.use_mfma ? launch_conv_mfma(a, NL.wp, NL.thr, NL.epi, s) : launch_conv_direct(a, s);
        break;
      }
      case PALQ_OP_CHANNEL_SHUFFLE: {
        palq_act iv = net->tensors[sp.src].d;
        if (sp.src == 0) iv.data = (void *)input;
        e = launch_channel_shuffle(view_of(&iv), view_of(&net->tensors[sp.dst].d), s);
        break;
      }
      case PALQ_OP_MAXPOOL: {
        palq_act iv = net->tensors[sp.src].d;
        if (sp.src == 0) iv.data = (void *)input;
        e = launch_maxpool(view_of(&iv), sp.pool_k, sp.pool_stride, sp.pool_pad,
                           view_of(&net->tensors[sp.dst].d), s);
        break;
      }
      case PALQ_OP_AVGSUM: {
        palq_act iv = net->tensors[sp.src].d;
        if (sp.src == 0) iv.data = (void *)input;
        e = launch_avgsum(view_of(&iv), NL.sums_out, s, NL.fc_planes_out, NL.fc_planes_n,
                          NL.fc_planes_out ? logits : nullptr, NL.fc_cout);
        break;
      }
      case PALQ_OP_FC:
        e = launch_fc(NL.fc_in, net->n, NL.fc_cin, NL.fc_w, sp.fc_out, logits, NL.fc_scratch, s, NL.fc_xmax,
                      NL.fc_planes_ready);
        break;
    }
    if (ev && e == hipSuccess) hipEventRecord(ev[i + 1], s);
  }
  if (e != hipSuccess) return net_fail(ctx, PALQ_ERR_DEVICE, std::string("forward: ") + hipGetErrorString(e));
  return PALQ_OK;
}
// PALQ_NET_GRAPH: replay the captured launch sequence when the call matches
// the one it was captured for, else capture it anew (the first forward runs
// eagerly, which also fills the launchers' per-kernel caches).
palq_status forward_dispatch(palq_ctx *ctx, palq_net *net, const void *input, int32_t *logits, const float *img,
                             float l, float u) {
  hipStream_t s = ctx->stream;
  if (!(net->flags & PALQ_NET_GRAPH)) return forward_impl(ctx, net, input, logits, img, l, u, s);
  if (!net->graph_warm) {
    net->graph_warm = true;
    return forward_impl(ctx, net, input, logits, img, l, u, s);
  }
  const bool same = net->graph_exec && net->g_input == input && net->g_img == img && net->g_logits == logits &&
                    net->g_l == l && net->g_u == u && net->g_stream == s;
  if (!same) {
    if (net->graph_exec) hipGraphExecDestroy(net->graph_exec);
    if (net->graph) hipGraphDestroy(net->graph);
    net->graph_exec = nullptr;
    net->graph = nullptr;
    // captured on a stream of the network's own (the caller's may be the
    // null stream, which cannot capture); the graph is launched on the
    // caller's stream
    hipError_t e = hipSuccess;
    if (!net->cap_stream) e = hipStreamCreateWithFlags(&net->cap_stream, hipStreamNonBlocking);
    if (e == hipSuccess) e = hipStreamBeginCapture(net->cap_stream, hipStreamCaptureModeThreadLocal);
    if (e != hipSuccess) return net_fail(ctx, PALQ_ERR_DEVICE, std::string("graph capture: ") + hipGetErrorString(e));
    const palq_status st = forward_impl(ctx, net, input, logits, img, l, u, net->cap_stream);
    hipGraph_t g = nullptr;
    e = hipStreamEndCapture(net->cap_stream, &g);
    if (st != PALQ_OK) {
      if (g) hipGraphDestroy(g);
      return st;
    }
    if (e != hipSuccess || !g) return net_fail(ctx, PALQ_ERR_DEVICE, std::string("graph capture: ") + hipGetErrorString(e));
    hipGraphExec_t x = nullptr;
    e = hipGraphInstantiate(&x, g, nullptr, nullptr, 0);
    if (e != hipSuccess) {
      hipGraphDestroy(g);
      return net_fail(ctx, PALQ_ERR_DEVICE, std::string("graph instantiate: ") + hipGetErrorString(e));
    }
    net->graph = g;
    net->graph_exec = x;
    net->g_input = input; net->g_img = img; net->g_logits = logits;
    net->g_l = l; net->g_u = u; net->g_stream = s;
  }
  const hipError_t e = hipGraphLaunch(net->graph_exec, s);
  return e == hipSuccess ? PALQ_OK : net_fail(ctx, PALQ_ERR_DEVICE, std::string("graph launch: ") + hipGetErrorString(e));
}
}  // namespace

palq_status palq_forward(palq_ctx *ctx, palq_net *net, const void *input, int32_t *logits) {
  if (!ctx || !net) return PALQ_ERR_ARG;
  if (net->ctx != ctx) return net_fail(ctx, PALQ_ERR_ARG, "network belongs to another context");
  if (!input || !logits) return net_fail(ctx, PALQ_ERR_ARG, "null input or logits");
  if (((uintptr_t)input & 15u) || ((uintptr_t)logits & 3u))
    return net_fail(ctx, PALQ_ERR_ARG, "input must be 16-byte and logits 4-byte aligned");
  if (ctx->device < 0) return PALQ_OK;
  hipSetDevice(ctx->device);
  return forward_dispatch(ctx, net, input, logits, nullptr, 0.f, 0.f);
}

palq_status palq_forward_image(palq_ctx *ctx, palq_net *net, const float *x, float l, float u, int32_t *logits) {
  if (!ctx || !net) return PALQ_ERR_ARG;
  if (net->ctx != ctx) return net_fail(ctx, PALQ_ERR_ARG, "network belongs to another context");
  if (!net->img_input)
    return net_fail(ctx, PALQ_ERR_ARG, "network input is not a signed 8-bit 3-channel image (one group)");
  if (!x || !logits) return net_fail(ctx, PALQ_ERR_ARG, "null x or logits");
  if (((uintptr_t)x & 3u) || ((uintptr_t)logits & 3u))
    return net_fail(ctx, PALQ_ERR_ARG, "x and logits must be 4-byte aligned");
  if (!std::isfinite(l) || !std::isfinite(u) || !(u > l) || !std::isfinite(u - l))
    return net_fail(ctx, PALQ_ERR_ARG, "need finite l < u with finite u - l");
  if (ctx->device < 0) return PALQ_OK;
  hipSetDevice(ctx->device);
  if (net->img_direct) return forward_dispatch(ctx, net, nullptr, logits, x, l, u);
  const hipError_t e = launch_quantize(x, l, u, nullptr, view_of(&net->input), ctx->stream);
  if (e != hipSuccess) return net_fail(ctx, PALQ_ERR_DEVICE, std::string("quantize: ") + hipGetErrorString(e));
  return forward_dispatch(ctx, net, net->img_codes, logits, nullptr, 0.f, 0.f);
}

const char *palq_net_layer_kernels(const palq_net *net, int32_t layer, int32_t image) {
  if (!net || (image != 0 && image != 1) || layer < -1 || layer >= (int32_t)net->layers.size()) return nullptr;
  if (layer == -1) return image ? net->img_label.c_str() : "";
  if (net->labels[image].size() != net->layers.size()) return "";  // validate-only network: nothing planned
  return net->labels[image][layer].c_str();
}

palq_status palq_net_tensor(const palq_net *net, int32_t id, palq_act *desc) {
  if (!net || !desc || id < 0 || id >= (int32_t)net->tensors.size() || !net->tensors[id].exists)
    return PALQ_ERR_ARG;
  if (net->tensors[id].kind == kLogits || id == 0) return PALQ_ERR_ARG;
  *desc = net->tensors[id].d;
  return PALQ_OK;
}

palq_status palq_net_layer_times(palq_net *net, float *ms, int32_t *forwards) {
  if (!net || !ms || !forwards) return PALQ_ERR_ARG;
  if (!(net->flags & PALQ_NET_TIMING)) return net_fail(net->ctx, PALQ_ERR_ARG, "network built without PALQ_NET_TIMING");
  hipSetDevice(net->ctx->device);
  while (net->pending_begin < net->pending_end) {
    accumulate_slot(net, net->pending_begin % kRing);
    net->pending_begin += 1;
  }
  for (size_t i = 0; i < net->ms.size(); ++i) ms[i] = (float)net->ms[i];
  *forwards = net->forwards;
  return PALQ_OK;
}

palq_status palq_net_reset_times(palq_net *net) {
  if (!net) return PALQ_ERR_ARG;
  if (!(net->flags & PALQ_NET_TIMING)) return PALQ_ERR_ARG;
  hipSetDevice(net->ctx->device);
  while (net->pending_begin < net->pending_end) {
    accumulate_slot(net, net->pending_begin % kRing);
    net->pending_begin += 1;
  }
  std::fill(net->ms.begin(), net->ms.end(), 0.0);
  net->forwards = 0;
  return PALQ_OK;
}

}  // extern "C"
