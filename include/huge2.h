/*
 * huge2.h -- C ABI of libhuge2: phase-decomposed transposed and dilated 2-D
 * convolution for AMD Instinct MI355X (gfx950), after HUGE^2 (Shi, Xu,
 * Yuan, Zhu, arXiv 1907.11210).
 *
 * What is computed
 *   conv2d_transpose: the transposed (fractionally strided) convolution of
 *     section 2.1.1 / Algorithm 1,
 *       y[n,k,oh,ow] = bias[k] + sum_{c,i,j,m,q} x[n,c,i,j] * w[c,k,m,q]
 *                      over oh = i*stride_h - pad_h + m*dil_h,
 *                           ow = j*stride_w - pad_w + q*dil_w,
 *     with oh in [0, h_out), h_out = (h-1)*stride_h - 2*pad_h
 *     + dil_h*(r-1) + out_pad_h + 1 (same for w).
 *   conv2d_dilated: the dilated convolution of section 2.1.1 / Algorithm 2
 *     (cross-correlation, zero padding),
 *       y[n,k,oh,ow] = bias[k] + sum_{c,m,q} x[n,c, oh*stride_h - pad_h + m*dil_h,
 *                                              ow*stride_w - pad_w + q*dil_w] * w[k,c,m,q],
 *     h_out = floor((h + 2*pad_h - dil_h*(r-1) - 1)/stride_h) + 1.
 *   Both then apply desc->activation elementwise (none, ReLU or tanh; see
 *   huge2_activation) before rounding to the output dtype.
 *
 * How (section 3): the kernel is decomposed into stride_h*stride_w phase
 * sub-kernels (section 3.1, Eq. 1-4); each phase is a dense convolution over
 * the un-inflated input, untangled into per-tap 1x1 convolutions that
 * accumulate as one implicit GEMM (section 3.2.1); the result is written
 * straight to the phase's disjoint, interleaved output positions (the
 * scatter of section 3.1), so no inserted zero is multiplied and no output
 * element is written twice.  A stride-1 dilated convolution is split the
 * same way into dil_h*dil_w phase views of the input (section 3.2.2).
 *
 * Conventions common to every entry point
 *   - All tensor pointers are DEVICE pointers owned by the caller, contiguous
 *     in the stated logical order, 16-byte aligned.  x and y must not alias.
 *   - Layout (HUGE2_NCHW or HUGE2_NHWC) applies to x and y.  Weights are
 *     always in the framework order given per entry point, whatever the
 *     activation layout.
 *   - dtype HUGE2_F32: x, w, y are float; MFMA in fp32.  HUGE2_BF16: x, w, y
 *     are bfloat16; products accumulate in fp32; y is rounded to nearest
 *     even.  bias is always float (nullable).
 *   - hip_stream is a hipStream_t (NULL = the default stream).  Work is
 *     enqueued asynchronously; the call returns after enqueue.
 *   - Every argument is validated before any HIP call.  On an error nothing
 *     is enqueued and y is untouched.  No C++ exception crosses the ABI.
 *   - Results for one plan are deterministic (fixed summation order, no
 *     atomics).
 */
#ifndef HUGE2_H
#define HUGE2_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  HUGE2_OK = 0,
  HUGE2_ERR_INVALID_ARG = 1, /* bad pointer, size, or descriptor field */
  HUGE2_ERR_UNSUPPORTED = 2, /* valid, but not implemented (e.g. dilated with stride > 1 and
                                out_pad != 0) */
  HUGE2_ERR_ALLOC = 3,       /* device or host allocation failed */
  HUGE2_ERR_HIP = 4          /* a HIP runtime call or kernel launch failed */
} huge2_status;

typedef enum { HUGE2_F32 = 0, HUGE2_BF16 = 1 } huge2_dtype;
typedef enum { HUGE2_NCHW = 0, HUGE2_NHWC = 1 } huge2_layout;
/* Elementwise function applied by the epilogue after the bias (the
 * generator's nonlinearities, with batch normalisation folded into w and
 * bias): y = act(op(x) + bias).  HUGE2_ACT_RELU: max(v, 0); HUGE2_ACT_TANH:
 * tanh(v).  Forward entry points only; the weight-gradient entry points
 * return HUGE2_ERR_UNSUPPORTED for any activation but HUGE2_ACT_NONE. */
typedef enum { HUGE2_ACT_NONE = 0, HUGE2_ACT_RELU = 1, HUGE2_ACT_TANH = 2 } huge2_activation;

/* Problem descriptor: the paper's Conv2DTranspose(I, K, O, s_m, s_n) and
 * Conv2DDilated(I, K, O, s_m, s_n) (Algorithms 1-2), extended with batch,
 * padding, output padding and both stride and dilation per axis. */
typedef struct {
  int32_t n, c_in, h, w;        /* input: batch, channels, height, width (all >= 1) */
  int32_t c_out, r, s;          /* output channels; kernel height r and width s (>= 1) */
  int32_t stride_h, stride_w;   /* >= 1 (the paper's s_m, s_n for the transposed conv) */
  int32_t pad_h, pad_w;         /* >= 0, symmetric */
  int32_t out_pad_h, out_pad_w; /* transposed only: 0 <= out_pad < max(stride, dil); 0 for dilated */
  int32_t dil_h, dil_w;         /* >= 1 (the paper's s_m, s_n for the dilated conv) */
  int32_t layout;               /* huge2_layout */
  int32_t dtype;                /* huge2_dtype */
  int32_t activation;           /* huge2_activation, applied after the bias (0: none) */
  /* Grouped convolution (0 or 1: none; PyTorch's groups): c_in and c_out
   * split into `groups` equal groups, output channel k (of group k /
   * (c_out/groups)) sums only over its group's input channels, and w holds
   * c_out/groups (transposed) or c_in/groups (dilated) channels on its
   * second axis.  groups = c_in is the depthwise convolution (a channel
   * multiplier c_out/c_in).  Grouped layers run on a direct kernel that
   * forms each output from its phase's taps (section 3.1) and its group's
   * channels, and their weight gradients on a direct per-plane kernel (see
   * the training section); grouped launches (huge2_group) take groups <= 1
   * only. */
  int32_t groups;
} huge2_conv_desc;

typedef struct huge2_plan huge2_plan; /* opaque */

/* Human-readable name of a status code (static storage; never NULL). */
const char* huge2_status_str(huge2_status status);

/* Output height/width of the operation described by desc: the loop bounds
 * of Algorithm 1 (transposed = 1: h_out = (h-1)*stride - 2*pad +
 * dil*(r-1) + out_pad + 1) and Algorithm 2 (transposed = 0: h_out =
 * floor((h + 2*pad - dil*(r-1) - 1)/stride) + 1), section 2.1.1, read as
 * the output range those definitions cover (the printed bounds are garbled).
 * Host only, no HIP call.  INVALID_ARG if the descriptor is invalid or the
 * output would be empty. */
huge2_status huge2_output_shape(const huge2_conv_desc* desc, int32_t transposed, int32_t* h_out,
                                int32_t* w_out);

/* The data gradient of a strided / dilated conv (section 3.2.3: the error
 * maps are carried back through the same kernel) is the transposed conv of
 * dy with the same weight array, stride, padding and dilation; several input
 * sizes h give one output size, and the output padding of that transposed
 * conv picks the right one.  For the strided conv described by conv_desc
 * (input h x w), writes the output padding (*op_h, *op_w) that makes the
 * transposed conv of its h_out x w_out output return exactly h x w.
 * Host only.  INVALID_ARG for an invalid descriptor or NULL outputs. */
huge2_status huge2_dgrad_output_padding(const huge2_conv_desc* conv_desc, int32_t* op_h,
                                        int32_t* op_w);

/* Build a reusable plan (the decomposition of section 3.1 done once per
 * layer): enumerates the phases, their kernel taps and border classes on the
 * host, allocates the plan's device buffers (packed weights and the work
 * list), copies the work list and runs on hip_stream the kernel that gathers
 * w into per-tap, K-contiguous sub-kernel blocks (section 3.2.1: the N x C
 * matrix for each kernel position), then waits for hip_stream.
 *   transposed = 1: w is [c_in][c_out/groups][r][s] (the paper's C x N x R x S,
 *                   section 4.2; PyTorch ConvTranspose2d order).
 *   transposed = 0: w is [c_out][c_in/groups][r][s] (PyTorch Conv2d order).
 * w is read only by work enqueued on hip_stream: it may be freed or changed
 * once that work has completed.  *out receives the plan (NULL on error).
 * A layer with fewer output tiles than compute units also gets a plan-owned
 * fp32 workspace of up to 8 x |y| elements (at most 256 MiB) for its K
 * slices; executes of one plan therefore share it: enqueue them on one
 * stream (or order them).
 * Errors: INVALID_ARG (descriptor, null out/w), UNSUPPORTED, ALLOC, HIP. */
huge2_status huge2_plan_create(huge2_plan** out, const huge2_conv_desc* desc, int32_t transposed,
                               const void* w, void* hip_stream);

/* Run a plan: y = op(x) (+ bias) -- Algorithm 1 or 2 (section 2.1.1)
 * computed by the phase decomposition of section 3.1-3.2.  x and y are laid
 * out per the plan's descriptor; bias is NULL or [c_out] float.  Enqueues on
 * hip_stream the plan's main kernel (the phase GEMM or one of its direct
 * forms, huge2_plan_kernel names it), preceded, when x is NCHW or its
 * channel count is not a multiple of 16 bytes and the main kernel reads a
 * channel-contiguous input, by a kernel that re-lays x out into the plan's
 * staging buffer.  A plan is immutable once created; two
 * executes of one plan that needs staging must not overlap (they share the
 * staging buffer).  Errors: INVALID_ARG (null plan/x/y, x == y), HIP (launch
 * failure). */
huge2_status huge2_plan_execute(const huge2_plan* plan, const void* x, const float* bias, void* y,
                                void* hip_stream);

/* The two halves of huge2_plan_execute, for callers that want to schedule or
 * time them separately.  huge2_plan_stage_input enqueues the re-layout of x
 * into the plan's staging buffer when the plan needs one (NCHW input, or a
 * channel count that is not a multiple of 16 bytes) and does nothing
 * otherwise.  huge2_plan_run_gemm enqueues the phase GEMM: it reads the
 * staging buffer when the plan stages (x may then be NULL), x otherwise.
 * Errors: INVALID_ARG (null plan or y, x NULL when needed, x == y), HIP. */
huge2_status huge2_plan_stage_input(const huge2_plan* plan, const void* x, void* hip_stream);
huge2_status huge2_plan_run_gemm(const huge2_plan* plan, const void* x, const float* bias, void* y,
                                 void* hip_stream);

/* 1 if plan_execute of this plan enqueues the input re-layout kernel, else 0
 * (host only; -1 for a NULL plan). */
int32_t huge2_plan_stages_input(const huge2_plan* plan);

/* Name of the main kernel a plan launches and its tile shape, e.g.
 * "phase_gemm2_kernel 64x128 w4 k2" (static storage owned by the plan,
 * valid until huge2_plan_destroy; "" for a NULL plan).  Host only. */
const char* huge2_plan_kernel(const huge2_plan* plan);

/* Release a plan and its device buffers.  Waits for the device to finish
 * work that may still use them.  NULL is accepted.  Errors: HIP. */
huge2_status huge2_plan_destroy(huge2_plan* plan);

/* One-shot transposed convolution (Algorithm 1 semantics, computed by the
 * phase decomposition): plan_create + plan_execute + stream-ordered release
 * of the plan's buffers.  w is [c_in][c_out][r][s].  desc->out_pad_* obey
 * 0 <= out_pad < max(stride, dil).  Errors as plan_create/plan_execute. */
huge2_status huge2_conv2d_transpose(const huge2_conv_desc* desc, const void* x, const void* w,
                                    const float* bias, void* y, void* hip_stream);

/* The one-shot transposed convolution for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc): the same computation and arguments as
 * huge2_conv2d_transpose, but every device buffer the call needs (the packed
 * sub-kernel weights, the work list, the input staging and the K-slice
 * partials) is carved from a static device array of 64 MiB that the library
 * holds on each GPU it runs on until the process ends; no hipMalloc,
 * hipFree or other allocating routine is called (host memory holds the
 * plan's description during the call, which waits for hip_stream as plan
 * creation does).  Every call on one GPU uses that GPU's same array: calls
 * that overlap on one GPU (other streams, other host threads) race and must
 * be ordered by the caller; calls on one stream are ordered already.  A
 * layer whose buffers exceed the 64 MiB returns HUGE2_ERR_UNSUPPORTED with y
 * untouched.  Errors otherwise as huge2_conv2d_transpose. */
huge2_status huge2_conv2d_transpose_noalloc(const huge2_conv_desc* desc, const void* x,
                                            const void* w, const float* bias, void* y,
                                            void* hip_stream);

/* One-shot dilated convolution (Algorithm 2 semantics; stride 1 is computed
 * by dil_h x dil_w phase views, stride > 1 by the same GEMM core over a
 * direct gather).  w is [c_out][c_in][r][s]; desc->out_pad_* must be 0. */
huge2_status huge2_conv2d_dilated(const huge2_conv_desc* desc, const void* x, const void* w,
                                  const float* bias, void* y, void* hip_stream);

/* ---- several convolutions of one input in one launch ------------------- */

/* A group runs the GEMM work of several plans that read the same input as
 * ONE kernel launch: e.g. the parallel branches of an atrous spatial
 * pyramid, each a dilated convolution of one feature map with its own
 * dilation (section 3.2.2 applied per branch).  The works of all plans are
 * listed together, image by image, and inside an image the costliest first
 * (the number of kernel taps a tile multiplies differs between border
 * classes and between dilations): the eight XCDs of the MI355X then each
 * work through contiguous images, whose input rows every branch shares in
 * that XCD's L2, and the compute units finish together.  Every output
 * element is computed as by huge2_plan_execute of its own plan: the same
 * tiles and taps, and with the plans' own kernel the same summation order
 * (bitwise equal results).  A list long enough for two workgroups on every
 * compute unit may run the 4-wave form of the pipelined 128 x 256 tile
 * instead (huge2_group_kernel names it), whose 64-byte K blocks sum the
 * products in another order: equal to rounding.
 *
 * huge2_group_create: plans[0 .. count) (1 <= count <= 8) must be plans
 * whose main kernel is the phase GEMM without a staging pass or a K split
 * (huge2_plan_kernel names "phase_gemm"; huge2_plan_stages_input is 0), with
 * equal input descriptors (n, c_in, h, w, layout, dtype), output channels,
 * kernel size, output size, activation and tile shape; they may differ in
 * stride, padding and dilation.  The group keeps pointers to the plans, which must
 * outlive it, and owns a device copy of the merged work list (copied on
 * hip_stream, which it then waits for).  Errors: INVALID_ARG (NULL out or
 * plans, count out of range), UNSUPPORTED (plans that cannot share a
 * launch), ALLOC, HIP. */
typedef struct huge2_group huge2_group;
huge2_status huge2_group_create(huge2_group** out, const huge2_plan* const* plans, int32_t count,
                                void* hip_stream);

/* Enqueue the group's launch on hip_stream: y[i] = op_i(x) (+ bias[i]) for
 * plan i.  x is the shared input (the plans' layout); y is an array of
 * count output pointers (none NULL or equal to x); bias is NULL or an array
 * of count pointers, each NULL or [c_out] float.  Executes of one group may
 * overlap (nothing is written but the outputs).  Errors: INVALID_ARG, HIP. */
huge2_status huge2_group_execute(const huge2_group* group, const void* x, const float* const* bias,
                                 void* const* y, void* hip_stream);

/* Name and tile shape of the kernel the group launches (owned by the group;
 * "" for NULL). */
const char* huge2_group_kernel(const huge2_group* group);

/* Release a group (its plans are untouched).  NULL is accepted.  Errors: HIP. */
huge2_status huge2_group_destroy(huge2_group* group);

/* ---- training: weight gradients (section 3.2.3) ------------------------- */

/* Back-propagation of a GAN updates the kernels from the output errors dy
 * (the gradient of the loss with respect to y, the forward output's shape):
 *   transposed conv (generator layer), w-shaped dw [c_in][c_out][r][s]:
 *     dw[c,k,m,q] = sum over (n, i, j) of x[n,c,i,j] * dy[n,k, i*stride_h - pad_h
 *                   + m*dil_h, j*stride_w - pad_w + q*dil_w], terms whose dy index
 *                   falls outside the output omitted -- the input correlated with
 *                   the error maps read with the stride;
 *   dilated / strided conv (discriminator layer), dw [c_out][c_in][r][s]:
 *     dw[k,c,m,q] = sum over (n, oh, ow) of dy[n,k,oh,ow] * x[n,c, oh*stride_h
 *                   - pad_h + m*dil_h, ow*stride_w - pad_w + q*dil_w], out-of-range
 *                   x omitted -- the error maps spread by the stride ("dilated
 *                   derivative maps") correlated with the input.
 * (The data gradients are the other form: dx of a transposed conv is the
 * strided conv of dy with the same w, and dx of a strided conv is the
 * transposed conv of dy; both are the entry points above.)
 * How: the large tensor (dy for the transposed conv, x for the strided
 * conv) is gathered onto the small tensor's pixel grid -- untangled copies,
 * as the paper's C copies of each derivative map: one per tap, or one per
 * (row phase, kernel column) with halo rows, shared by the taps that differ
 * only in their row shift -- and the gradient of all taps is then one dense
 * MFMA GEMM over pixels with
 * no zero products (its columns are the (channel, tap) pairs, dw's own
 * order), accumulated in fp32 over K slices and chunks of images in a fixed
 * order and rounded once to the dtype.
 * Grouped layers (groups > 1; dw is [c_in][c_out/groups][r][s] or
 * [c_out][c_in/groups][r][s]): the sums above run only over channel pairs of
 * one group.  Each weight plane then joins one input map to one error map --
 * the depthwise form of section 3.2.3, an outer product of two maps summed
 * over the pixels -- and is summed directly in fp32 (one workgroup per plane
 * and run of 16 taps, a fixed reduction order), with no workspace.
 * Layout: NCHW only (HUGE2_NHWC returns HUGE2_ERR_UNSUPPORTED).  dtype as
 * above: x, dy and dw share it; accumulation is fp32 for both dtypes. */
typedef struct huge2_wgrad_plan huge2_wgrad_plan;

/* Build a weight-gradient plan for desc (the forward layer's descriptor;
 * transposed selects the layer type).  Allocates the per-plan workspace
 * (none for grouped layers): the staged operands of one chunk of images
 * (the chunk is sized so they stay under 256 MiB; at least one image) and,
 * unless one K slice covers the whole batch, the fp32 gradient slices (at
 * most 32 MiB).  No HIP
 * work is enqueued.  Errors: INVALID_ARG (NULL out/desc, invalid
 * descriptor), UNSUPPORTED (NHWC; byte extents of 2^31 or more), ALLOC. */
huge2_status huge2_wgrad_plan_create(huge2_wgrad_plan** out, const huge2_conv_desc* desc,
                                     int32_t transposed);

/* Enqueue dw for input x and output error dy (device pointers, NCHW, the
 * plan's dtype) on hip_stream; dw must not alias x or dy.  Calls on one
 * plan share its workspace: enqueue them on one stream (or order them).
 * Errors: INVALID_ARG (NULL plan/pointer, aliasing), HIP. */
huge2_status huge2_wgrad_execute(const huge2_wgrad_plan* plan, const void* x, const void* dy,
                                 void* dw, void* hip_stream);

/* Release a weight-gradient plan; waits for the device first.  NULL is
 * accepted.  Errors: HIP. */
huge2_status huge2_wgrad_plan_destroy(huge2_wgrad_plan* plan);

/* One-shot forms: plan_create + execute + destroy (synchronises the
 * stream before releasing the workspace). */
huge2_status huge2_conv2d_transpose_wgrad(const huge2_conv_desc* desc, const void* x,
                                          const void* dy, void* dw, void* hip_stream);
huge2_status huge2_conv2d_dilated_wgrad(const huge2_conv_desc* desc, const void* x,
                                        const void* dy, void* dw, void* hip_stream);

/* ---- introspection (host only, no HIP call) ---------------------------- */

/* One rectangle of a box of phases with a constant set of kernel taps.
 * Output positions: oh = phase_h + out_step_h * qh for every phase_h in
 * [phase0_h, phase0_h + nphase_h) and qh in [q0_h, q0_h + qn_h), likewise
 * ow; every image n in [0, desc.n).  Tap t of the segment (t in
 * [tap_begin, tap_begin + tap_count) of the tap list) reads input row
 *   ih = in0_h + in_dphase_h * (phase_h - phase0_h) + in_step_h * qh + taps[t].off_h
 * (likewise iw) with kernel tap (taps[t].kh, taps[t].kw).  Transposed convs
 * use one phase per segment (each phase has its own sub-kernel); stride-1
 * dilated convs group the phase views that share a shape.  A segment with
 * tap_count 0 is an output region no input reaches (it holds the bias). */
typedef struct {
  int32_t phase0_h, phase0_w, nphase_h, nphase_w;
  int32_t out_step_h, out_step_w;
  int32_t q0_h, q0_w, qn_h, qn_w;
  int32_t in0_h, in0_w, in_dphase_h, in_dphase_w, in_step_h, in_step_w;
  int32_t tap_begin, tap_count;
} huge2_segment;

typedef struct {
  int32_t kh, kw;       /* kernel tap */
  int32_t off_h, off_w; /* input offset added to in_base + in_step * q */
} huge2_tap;

/* The decomposition a plan for desc would use.  Fills up to seg_cap
 * segments and tap_cap taps; *n_segs / *n_taps receive the full counts (call
 * with caps 0 to size the arrays).  class_split: 1 splits every phase into
 * border classes, so that each segment reads only in-range inputs; 0 keeps
 * one segment per phase group with all of its taps (out-of-range reads then
 * contribute zero); 2 chooses per phase group whichever issues fewer
 * tile-taps for the plan's tile height.  A plan uses 0 or 2, whichever a
 * model of its schedule on the MI355X's compute units finishes first. */
huge2_status huge2_plan_describe(const huge2_conv_desc* desc, int32_t transposed,
                                 int32_t class_split, huge2_segment* segs, int32_t seg_cap,
                                 int32_t* n_segs, huge2_tap* taps, int32_t tap_cap,
                                 int32_t* n_taps);

/* Counts for a descriptor: structural non-zero multiply-adds (products of an
 * input element and a kernel tap that land on an output element: no inserted
 * zero, no padding, no cropped position) and the multiply-adds the plan's
 * GEMM tiles actually issue (including tile padding). */
huge2_status huge2_plan_macs(const huge2_conv_desc* desc, int32_t transposed, int64_t* nonzero_macs,
                             int64_t* issued_macs);

#ifdef __cplusplus
}
#endif
#endif /* HUGE2_H */
