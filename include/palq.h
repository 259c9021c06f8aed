/*
 * palq.h -- C ABI of the PalQuant inference library for AMD MI355X (gfx950).
 *
 * PalQuant (parallel low-precision quantisation) runs a high-precision
 * network as G parallel groups of B-bit convolutions (Section 4.1), with a
 * cyclic permutation of the groups between layers (Section 4.2, Eq. 6-8).
 * This library computes the integer inference path of such a network on one
 * GPU: quantise (Eq. 2), grouped B-bit convolution with int32 accumulation
 * (Eq. 1 per group), a fixed-point requantisation with ReLU, and the cyclic
 * permutation applied as the write address of the result.
 *
 * Conventions for every call
 *  - Tensor and parameter pointers are DEVICE pointers owned by the caller
 *    unless a comment says "host".  The library never frees them.
 *  - Calls are asynchronous on the context's stream.  All argument checks
 *    happen on the host before anything is enqueued: a call that returns an
 *    error other than PALQ_ERR_DEVICE has written nothing.  Device faults
 *    surface on a later call or on palq_sync.
 *  - No call throws or aborts across the ABI.  palq_last_error() gives a
 *    human-readable reason for the last failing call on that context.
 *  - A context is used by one host thread at a time.
 *  - A context created with device = -1 is "validate only": every call checks
 *    its arguments exactly as on a GPU and then returns without device work.
 *
 * Packed code layout (activations and filters)
 *  A tensor [N][H][W][G][C^] of b-bit codes is stored NHWC, group-major
 *  (channel g*C^ + j, the [N, G, C^, H, W] view of Section 4.2).  Each
 *  (pixel, group) row of C^ codes occupies palq_row_bytes(C^, b) bytes and
 *  rows follow each other with no gap; a pixel is G rows.  That is layout
 *  PALQ_LAYOUT_PIXEL.  PALQ_LAYOUT_GROUP stores the same rows as
 *  [G][N][H][W]: all of group 0's rows in pixel order, then group 1's, ...
 *  (a group's rows of consecutive pixels are adjacent, so one group's tile
 *  of pixels is one contiguous run).  Both take palq_act_bytes() bytes.
 *   - b in {2, 4, 8}: code j sits at bits [b*j, b*j + b) of the row read as
 *     one little-endian bit string; the row is padded with zero bits to a
 *     multiple of 32 bits.
 *   - b = 6: stored as b = 8 (code j in bits 0-5 of byte j, bits 6-7 zero),
 *     for dense 6-bit baselines.
 *   - b = 3: the row is cut into chunks of 32 codes (the last one padded with
 *     zero codes), 12 bytes each.  In a chunk, bytes 0-7 are a little-endian
 *     64-bit field holding bits 0-1 of code j at bits [2j, 2j+2); bytes 8-11
 *     are a little-endian 32-bit field holding bit 2 of code j at bit
 *     2*(j & 15) + (j >> 4) (codes 0-15 at the even bits, 16-31 at the odd
 *     bits).
 *  Signed codes are b-bit two's complement, unsigned codes are plain binary.
 *  Padding bits are written as zero and ignored when read.
 *  A filter [G][C^out][kh][kw][C^in] has the layout of an activation tensor
 *  with N = G*C^out, H = kh, W = kw and one group of C^in codes.
 */
#ifndef PALQ_H
#define PALQ_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t palq_status;
#define PALQ_OK 0
#define PALQ_ERR_ARG (-1)         /* malformed or inconsistent arguments        */
#define PALQ_ERR_UNSUPPORTED (-2) /* well formed but outside what is built      */
#define PALQ_ERR_OVERFLOW (-3)    /* the int32 accumulator bound could be broken */
#define PALQ_ERR_DEVICE (-4)      /* HIP runtime error                          */
#define PALQ_ERR_NOMEM (-5)       /* device or host allocation failed           */

typedef struct palq_ctx palq_ctx;
typedef struct palq_net palq_net;

/* An activation tensor: n x h x w pixels of `groups` rows of ch_per_group
 * codes, `bits` in {2, 3, 4, 8}.  data: device, palq_act_bytes() bytes.
 * layout: PALQ_LAYOUT_PIXEL (0, what a zeroed descriptor holds) or
 * PALQ_LAYOUT_GROUP (see the packed code layout above); every call takes
 * either, and the tensors of one call may mix them. */
#define PALQ_LAYOUT_PIXEL 0
#define PALQ_LAYOUT_GROUP 1
typedef struct {
  int32_t n, h, w;
  int32_t groups, ch_per_group;
  int32_t bits;
  int32_t is_signed;
  int32_t layout;
  void *data;
} palq_act;

/* A grouped filter: groups x cout_pg output channels, each a kh x kw x
 * cin_pg block of signed `bits`-bit codes (bits in {2, 3, 4, 8}).
 * data: device, packed as described above. */
typedef struct {
  int32_t groups, cout_pg, cin_pg, kh, kw, bits;
  const void *data;
} palq_filter;

/* Per-output-channel fixed-point requantisation, arrays of groups*cout_pg
 * int32 on the device, indexed by the convolution's own output channel
 * g*cout_pg + k (before the cyclic permutation moves it):
 *   q = clamp(floor((t * mult + 2^(shift-1)) / 2^shift), 0, 2^out_bits - 1)
 * with t = acc + bias + residual (below).  The clamp at 0 is the fused ReLU.
 * The result is exact for mult in [0, 2^31), shift in [1, 62], |bias| < 2^30
 * and |res_mult| < 2^15 (outside that range the output is unspecified but
 * no memory outside the output tensor is touched).  bias may be NULL (0).
 * out_bits in {2, 3, 4, 8}; output codes are unsigned.  The arrays (and
 * res_mult below) must be 16-byte aligned. */
typedef struct {
  const int32_t *mult;
  const int32_t *shift;
  const int32_t *bias;
  int32_t out_bits;
} palq_requant;

/* Shortcut added to t in int64 before requantisation, at the DESTINATION
 * channel of the cyclic permutation.  At most one of the two kinds:
 *  - identity: t += res_mult[c] * identity[pixel, dest channel], where
 *    `identity` has the output's shape (any unsigned bits) and res_mult is
 *    indexed like the requant arrays (device, groups*cout_pg int32);
 *  - projection: t += the int32 accumulator, at the destination channel, of
 *    the 1x1 grouped convolution of proj_in with proj_w at stride
 *    proj_stride, pad 0 (proj_w: same groups and cout_pg as the main filter,
 *    kh = kw = 1; proj_in: unsigned codes, groups = proj_w->groups). */
typedef struct {
  const palq_act *identity;
  const int32_t *res_mult;
  const palq_act *proj_in;
  const palq_filter *proj_w;
  int32_t proj_stride;
} palq_residual;

/* ---------------------------------------------------------------- context */

/* Creates a context on HIP device `device` (or -1: validate only) that
 * enqueues on `hip_stream` (a hipStream_t; NULL = the null stream).
 * Returns PALQ_ERR_DEVICE when the device cannot be used. */
palq_status palq_create(int32_t device, void *hip_stream, palq_ctx **out);
void palq_destroy(palq_ctx *ctx);
/* Later calls enqueue on hip_stream.  The new stream first waits for the
 * work already queued on the old one (which may still read context memory
 * that later calls reuse). */
palq_status palq_set_stream(palq_ctx *ctx, void *hip_stream);
/* Matrix-core format of 2- and 3-bit grouped convolutions (Section 4.1):
 * with enable = 1 (the default; environment PALQ_CONV_FP4=0 starts a context
 * at 0) a layer whose accumulator bound sum |w| |x| stays below 2^23 runs on
 * the FP4 (E2M1) matrix cores if it is a 2-bit layer, on the FP6 (E2M3)
 * matrix cores if it is a 3-bit layer with 3-bit outputs, 64-channel blocks
 * and no shortcut, where its fp32 accumulator is exact; with 0 every layer
 * runs on int8.  Results are identical either way.  Applies to
 * palq_group_conv calls and networks created after the call.
 * PALQ_ERR_ARG: enable not 0 or 1. */
palq_status palq_set_conv_fp4(palq_ctx *ctx, int32_t enable);
/* Execution of wide grouped convolutions as the bit-level decomposition of
 * Section 3.2 (Eq. 4), the baseline PalQuant is set against (Section 5.2,
 * Table 2): with enable = 1 a layer with unsigned M-bit inputs, M-bit
 * weights and M-bit outputs, M in {4, 6, 8}, 64-channel blocks and an
 * optional M-bit identity or projection shortcut splits every code into
 * M / 2 2-bit chunks and runs the (M / 2)^2 chunk products of each MAC on
 * the FP4 matrix cores, shifted by 4^(i+j) and summed exactly
 * ("conv_bitdecomp_kernel"), where the accumulator bounds allow it; with 0
 * (the default) such layers run directly on int8.  Results are identical
 * either way.  Applies to palq_group_conv calls and networks created after
 * the call.  PALQ_ERR_ARG: enable not 0 or 1. */
palq_status palq_set_conv_bitdecomp(palq_ctx *ctx, int32_t enable);
/* Waits for all work on the context's stream; reports deferred device errors. */
palq_status palq_sync(palq_ctx *ctx);
/* Reason for the last failed call on ctx; owned by ctx, valid until its next call. */
const char *palq_last_error(const palq_ctx *ctx);
/* Library build string (host; static storage). */
const char *palq_version(void);

/* Bytes of one packed row of `codes` codes at `bits` bits (-1 if invalid). */
int64_t palq_row_bytes(int32_t codes, int32_t bits);
/* Bytes of a packed activation tensor (-1 if the descriptor is invalid). */
int64_t palq_act_bytes(const palq_act *a);

/* ------------------------------------------------------------ data layout */

/* Packs one code per byte, [n][h][w][groups*ch_per_group] (int8 for signed,
 * uint8 for unsigned codes), into `out`'s layout.  Codes outside the b-bit
 * range are truncated to their low b bits. */
palq_status palq_pack(palq_ctx *ctx, const void *codes, const palq_act *out);
/* The inverse: one code per byte, signed codes sign-extended. */
palq_status palq_unpack(palq_ctx *ctx, const palq_act *in, void *codes);

/* ------------------------------------------------------------ hot path */

/* Uniform quantiser, Section 3.2 Eq. 2, elementwise over an fp32 NHWC tensor
 * x of out's shape: d = x - l, r = u - l, t = d / r (IEEE fp32, correctly
 * rounded), t = min(t, 1), t = (t >= 0 ? t : 0) (NaN -> 0),
 * q = rint(t * (2^b - 1)) with ties to even, and q - 2^(b-1) for signed
 * codes.  If l or u is NaN both are taken as the min and max of the non-NaN
 * elements of x (computed on the device); range_out (device, 2 floats,
 * nullable) receives the l and u used.  Host check: u > l and u - l finite
 * when both are given.  If the calibrated range is empty or degenerate the
 * output is all zero codes (the minimum code when signed). */
palq_status palq_quantize(palq_ctx *ctx, const float *x, float l, float u, const palq_act *out,
                          float *range_out);

/* One PalQuant layer: G parallel B-bit convolutions (Section 4.1; Eq. 1 per
 * group), int32 accumulation, then requantisation (palq_requant) with the
 * optional shortcut (palq_residual), and the cyclic permutation of Eq. 8
 * applied `shuffle_steps` times as the write address: the result of source
 * group g is stored in group (g + shuffle_steps) mod G.
 *   in  : unsigned codes of 2, 3, 4, 6 or 8 bits, or signed 8-bit codes;
 *         groups == w->groups, ch_per_group == w->cin_pg
 *   out : n x ho x wo, groups == w->groups, ch_per_group == w->cout_pg,
 *         bits == rq->out_bits, unsigned; ho = (h + 2 pad - kh)/stride + 1
 *   acc_dump (nullable, 16-byte aligned): int32 [n][ho][wo][groups*cout_pg], the sum of all
 *         products that land in each output channel (destination order:
 *         the permuted main accumulator plus any projection accumulator).
 * PALQ_ERR_OVERFLOW when K*max|code|*max|weight| (K = kh*kw*cin_pg), plus
 * the same bound of the projection product, reaches 2^26 for 2-bit inputs
 * or 2^30 for wider ones; a projection input is unsigned codes.  out
 * must not
 * overlap any input.  Every call prepacks the filter again, into context
 * memory that it grows (allocating) when a call needs more than any before;
 * it never synchronises.  A loop over one layer plans it once instead
 * (palq_conv_plan_create) and runs the plan (palq_conv_run). */
palq_status palq_group_conv(palq_ctx *ctx, const palq_act *in, const palq_filter *w, int32_t stride,
                            int32_t pad, const palq_requant *rq, const palq_residual *res,
                            int32_t shuffle_steps, const palq_act *out, int32_t *acc_dump);

/* palq_group_conv for callers that cannot allocate device memory: code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  Same arguments, checks, arithmetic and results as
 * palq_group_conv, but the layer's prepacked filter and requant constants go
 * into a static device buffer of PALQ_NOALLOC_SCRATCH_BYTES that the library
 * holds on every GPU it runs on (until the process ends) instead of context
 * memory, and the call allocates, frees and synchronises nothing.  Every
 * call on one GPU shares that buffer and it keeps the last call's contents:
 * calls on one stream are ordered, calls that overlap on one GPU (other
 * streams, contexts or host threads) race.  PALQ_ERR_UNSUPPORTED (nothing
 * written) when the prepacked filter and constants of the layer exceed the
 * buffer; PALQ_ERR_DEVICE when the buffer is unavailable on this device. */
#define PALQ_NOALLOC_SCRATCH_BYTES (16 << 20)
palq_status palq_group_conv_noalloc(palq_ctx *ctx, const palq_act *in, const palq_filter *w, int32_t stride,
                                    int32_t pad, const palq_requant *rq, const palq_residual *res,
                                    int32_t shuffle_steps, const palq_act *out, int32_t *acc_dump);

/* A planned layer: the filter, the requant and shortcut parameters of one
 * palq_group_conv layer, prepacked into the matrix-core operand order with
 * its requant constants and its kernel chosen, once, for repeated runs. */
typedef struct palq_conv_plan palq_conv_plan;

/* Plans the layer palq_group_conv computes (same arguments and checks,
 * Section 4.1 / Eq. 1 per group, Eq. 8 as the write address): copies w,
 * rq's arrays, res->res_mult and res->proj_w into device memory the plan
 * owns, prepacks the filter, computes the requant constants and reads back
 * which epilogue applies (this call synchronises the context's stream once).
 * Only the shapes, bits, signs and layouts of in, out, res->identity and res->proj_in
 * are used; their data pointers are ignored.  The caller may free the
 * parameter arrays once this returns.  A validate-only context returns a
 * plan that runs nothing.  Errors as palq_group_conv; PALQ_ERR_NOMEM. */
palq_status palq_conv_plan_create(palq_ctx *ctx, const palq_act *in, const palq_filter *w, int32_t stride,
                                  int32_t pad, const palq_requant *rq, const palq_residual *res,
                                  int32_t shuffle_steps, const palq_act *out, palq_conv_plan **plan);
/* Runs a plan on device tensors of the planned shapes: in, out, res_in (the
 * identity shortcut's codes or the projection input, as planned; NULL when
 * the plan has no shortcut) and acc_dump (nullable; as in palq_group_conv),
 * all 16-byte aligned.  Enqueues the planned kernels on the context's
 * stream and nothing else: no allocation, no synchronisation, no host copy,
 * so it may be captured into a HIP graph.  PALQ_ERR_ARG for a plan of
 * another context, null, misaligned or overlapping pointers, or a shortcut
 * input that does not match the plan. */
palq_status palq_conv_run(palq_ctx *ctx, const palq_conv_plan *plan, const void *in, const void *res_in, void *out,
                          int32_t *acc_dump);
/* Frees a plan (waits for device work that still reads it). */
void palq_conv_plan_destroy(palq_conv_plan *plan);
/* The kernel family a plan runs without an accumulator dump (static host
 * string, e.g. "conv_fp4_kernel"; "" for a validate-only plan; NULL
 * for a null plan). */
const char *palq_conv_plan_kernels(const palq_conv_plan *plan);

/* The cyclic permutation of Section 4.2 (Eq. 6-8) on its own:
 * out[pixel, (g + steps) mod G, :] = in[pixel, g, :], any integer steps.
 * in and out have the same shape and bits and must not overlap. */
palq_status palq_cyclic_shuffle(palq_ctx *ctx, const palq_act *in, int32_t steps,
                                const palq_act *out);

/* The cyclic shuffle module of Section 4.2 (Eq. 9-10), Z = X + Conv1x1(Y)
 * with Y = CyclicPermute(X) (Eq. 8, one step), as an integer layer:
 *   t[p, j, k] = sum_c w[j][k][c] * in[p, (j - 1) mod G, c] + bias[j*C + k]
 *                + res_mult[j*C + k] * in[p, j, k]
 *   out[p, j, k] = clamp(floor((t M + 2^(sh-1)) / 2^sh), 0, 2^out_bits - 1)
 * with M, sh = rq->mult, rq->shift [j*C + k].  Every per-channel array is
 * indexed by the module's output channel j*C + k.
 *   in  : unsigned codes of 2, 3 or 4 bits, G groups of C codes
 *   w   : 1x1 filter, groups G, cout_pg == cin_pg == C, bits == in bits
 *   out : in's n, h, w, groups and C; bits == rq->out_bits (2, 3, 4 or 8)
 *   res_mult: device int32 [G*C], |res_mult| < 2^15
 * Device pointers, caller-owned; out must not overlap in.  Runs as one
 * grouped 1x1 layer that stores its branch one group on with the identity
 * shortcut from in, its per-group parameters rotated by one group into
 * context-owned memory first (asynchronously, on the context stream).
 * Errors as palq_group_conv. */
palq_status palq_shuffle_module(palq_ctx *ctx, const palq_act *in, const palq_filter *w,
                                const palq_requant *rq, const int32_t *res_mult, const palq_act *out);

/* Channel shuffle across the groups of each pixel (the per-stage channel
 * shuffle of Section 4.3 and Table 3; the [G][C] channel matrix transposed
 * to [C][G]): out channel o = g*C + c takes in channel (o mod G)*C + o / G.
 * in and out have the same shape and bits and must not overlap. */
palq_status palq_channel_shuffle(palq_ctx *ctx, const palq_act *in, const palq_act *out);

/* k x k max pool with stride and zero-area padding (max over the in-image
 * part of each window) on unsigned codes; out has in's groups and bits. */
palq_status palq_maxpool(palq_ctx *ctx, const palq_act *in, int32_t k, int32_t stride, int32_t pad,
                         const palq_act *out);

/* Global average pool kept as the exact integer sum over h x w of unsigned
 * codes: out int32 [n][groups*ch_per_group]. */
palq_status palq_avgsum(palq_ctx *ctx, const palq_act *in, int32_t *out);

/* Fully connected layer on integer features (Eq. 1):
 * logits[i][o] = sum_c x[i][c] * w[o][c], x int32 [n][cin], w int8
 * [cout][cin], logits int32 [n][cout].  The sum is formed modulo 2^32, so a
 * logit is exact whenever its true value fits int32. */
palq_status palq_fc(palq_ctx *ctx, const int32_t *x, int32_t n, int32_t cin, const int8_t *w,
                    int32_t cout, int32_t *logits);

/* ------------------------------------------------------------ networks */

#define PALQ_OP_CONV 1
#define PALQ_OP_MAXPOOL 2
#define PALQ_OP_AVGSUM 3
#define PALQ_OP_FC 4
#define PALQ_OP_SHUFFLE_MODULE 5
#define PALQ_OP_CHANNEL_SHUFFLE 6

#define PALQ_NET_KEEP_ALL 1 /* every tensor keeps its own buffer (for inspection) */
#define PALQ_NET_TIMING 2   /* record a HIP event pair around every layer      */
#define PALQ_NET_GRAPH 4    /* replay forwards from a captured HIP graph: the
                             * first forward runs eagerly, later ones capture
                             * the launch sequence once per (input, logits, l,
                             * u, stream) and replay it; input contents may
                             * change between calls.  Not with PALQ_NET_TIMING. */
#define PALQ_NET_PIXEL_LAYOUT 8 /* keep every tensor in PALQ_LAYOUT_PIXEL; by
                                 * default a conv, channel shuffle or max pool
                                 * output of several groups whose every reader
                                 * takes it with those groups is stored in
                                 * PALQ_LAYOUT_GROUP (palq_net_tensor reports
                                 * each tensor's layout) */

/* One layer of a network.  Tensor ids: 0 is the network input; each layer
 * writes a new id `dst` larger than every id before it.  Every pointer in
 * a layer is a host or device pointer (any address HIP's default copy kind
 * accepts) to data that palq_net_create copies into the network's own pool
 * before it returns (the caller may free it afterwards):
 *   w.data / proj_w.data: packed filter bytes; mult/shift/bias/res_mult:
 *   int32 [groups*cout_pg]; fc_w: int8 [fc_out][cin].
 *  PALQ_OP_CONV    src (codes, viewed as w.groups rows of w.cin_pg codes; a
 *                  tensor may be re-grouped when its rows have no padding),
 *                  w, stride, pad, mult/shift/bias (bias nullable), out_bits,
 *                  shuffle_steps; optional identity shortcut res_src (>= 0)
 *                  with res_mult, or projection proj_src (>= 0) with proj_w
 *                  and proj_stride.  Same arithmetic as palq_group_conv.
 *  PALQ_OP_SHUFFLE_MODULE src, w (1x1, cout_pg == cin_pg), mult/shift/bias
 *                  (bias nullable), out_bits, res_mult: the cyclic shuffle
 *                  module of palq_shuffle_module (the other conv fields are
 *                  ignored).
 *  PALQ_OP_CHANNEL_SHUFFLE src -> the same shape (palq_channel_shuffle).
 *  PALQ_OP_MAXPOOL src, pool_k, pool_stride, pool_pad.
 *  PALQ_OP_AVGSUM  src -> int32 sums [n][channels].
 *  PALQ_OP_FC      src (an AVGSUM output), fc_w, fc_out -> int32 logits.
 * The last layer must be PALQ_OP_FC; its output is forward's logits. */
typedef struct {
  int32_t op;
  int32_t src, dst;
  palq_filter w;
  int32_t stride, pad;
  const int32_t *mult, *shift, *bias;
  int32_t out_bits;
  int32_t shuffle_steps;
  int32_t res_src;
  const int32_t *res_mult;
  int32_t proj_src;
  palq_filter proj_w;
  int32_t proj_stride;
  int32_t pool_k, pool_stride, pool_pad;
  const int8_t *fc_w;
  int32_t fc_out;
} palq_layer;

/* Validates the layer list against the input descriptor (shape, bits, sign;
 * its data pointer is ignored), plans buffers, copies all parameters to the
 * device and returns a network bound to ctx.  flags: PALQ_NET_*. */
palq_status palq_net_create(palq_ctx *ctx, const palq_act *input, const palq_layer *layers,
                            int32_t n_layers, int32_t flags, palq_net **out);
void palq_net_destroy(palq_net *net);

/* Runs the network on `input` (device, packed as the input descriptor says)
 * and writes logits (device, int32 [n][fc_out]).  Asynchronous. */
palq_status palq_forward(palq_ctx *ctx, palq_net *net, const void *input, int32_t *logits);

/* The quantiser of Section 3.2 Eq. 2 (as palq_quantize with fixed l, u and
 * signed 8-bit codes) followed by palq_forward, for a network whose input
 * descriptor is a signed 8-bit image with one group of 3 channels.  x:
 * device fp32 [n][h][w][3] of that shape, 4-byte aligned.  Results are
 * identical to palq_quantize into an input tensor and palq_forward on it;
 * where the first layer copies its input with a zero border the codes are
 * written straight into that copy (no separate input tensor or copy).
 * Errors: PALQ_ERR_ARG for another input format, null or misaligned
 * pointers, or l, u not finite with u > l.  Asynchronous. */
palq_status palq_forward_image(palq_ctx *ctx, palq_net *net, const float *x, float l, float u, int32_t *logits);

/* Descriptor (with device data pointer) of tensor `id` after a forward pass.
 * Conv/maxpool outputs are packed codes in the layout the descriptor names
 * (see PALQ_NET_PIXEL_LAYOUT; palq_unpack reads either); an AVGSUM output
 * is reported with bits = 32 (int32 values, one per channel, h = w = 1).
 * Valid for every id only with PALQ_NET_KEEP_ALL; otherwise buffers are
 * reused between layers. */
palq_status palq_net_tensor(const palq_net *net, int32_t id, palq_act *desc);

/* Algorithmic work of one forward pass: 2 * multiply-accumulates of every
 * conv (main and projection) and FC layer (host). */
int64_t palq_net_ops(const palq_net *net);

/* The kernels a forward pass launches for layer `layer`, as the library's
 * own selection rules pick them at create time (host string owned by net,
 * valid until palq_net_destroy): e.g. "conv_fp4_kernel" or
 * "quantize_pad4_kernel + stem_pool_kernel"; "" for a layer that an earlier
 * layer's launch already covers (a max pool fused into the stem) and for
 * every layer of a validate-only network.  image = 0: palq_forward,
 * 1: palq_forward_image; layer = -1 names forward_image's quantiser pass
 * into a buffer of its own ("" when the codes go straight into the stem's
 * zero-border input).  NULL for a null net, a bad index or image. */
const char *palq_net_layer_kernels(const palq_net *net, int32_t layer, int32_t image);

/* With PALQ_NET_TIMING: per-layer device time of every forward since the
 * last reset, summed, in milliseconds (host array of n_layers floats), and
 * the number of forwards it covers.  Synchronises the stream. */
palq_status palq_net_layer_times(palq_net *net, float *ms, int32_t *forwards);
palq_status palq_net_reset_times(palq_net *net);

#ifdef __cplusplus
}
#endif
#endif /* PALQ_H */
