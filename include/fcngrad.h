/*
 * fcngrad — one GPU's share of a data-parallel training step of a fully
 * convolutional encoder-decoder in fp16 (Laanait et al., "Exascale Deep
 * Learning for Scientific Inverse Problems", arXiv 1909.11150), for AMD
 * Instinct MI355X (gfx950).
 *
 * The step has two halves:
 *   1. the three convolution passes of every layer — forward, gradient with
 *      respect to the kernel, gradient with respect to the input (Section
 *      5.2: the passes counted by the factor 3 in the Sustained and Peak
 *      performance equations; the operation count of each is the
 *      direct-convolution count OPS_conv of that section) — plus the
 *      transposed convolution of the decoder (Section 6.2, Figure workflow
 *      (B): encoder-decoder network) and the ReLU after each layer (Section
 *      6.2, Neural Network Architecture), fused into the convolutions;
 *   2. the gradient path between back-propagation and the optimizer: the
 *      weight gradients are fused into contiguous group buffers (Section
 *      4.2, Grouping: only complete groups are fused into one message), the
 *      loss scale is removed and overflow is detected (Section 6.2, Model
 *      Implementation: loss scaling keeps values inside the float16 range),
 *      and the fp32 gradients are scattered back to per-tensor buffers.
 * On more than one GPU a sum-allreduce of each packed group sits between
 * grad_group_pack and grad_unscale_check; this library is the per-GPU part.
 *
 * Conventions (all entry points)
 *   - fp16 data is passed as uint16_t bit patterns (IEEE binary16).
 *     Activations are NHWC. Convolution weights are KRSC (out channel,
 *     kernel row, kernel column, in channel). Transposed-convolution weights
 *     are C_in x R x S x C_out. Convolution is cross-correlation (no flip);
 *     padding is symmetric zero padding; forward output size is
 *     P = (H + 2*pad_h - R)/stride_h + 1 (floor), likewise Q.
 *   - Every device pointer (x, w, y, gate, ws, group buffers, flags, segment
 *     targets) is owned by the caller. The library never allocates or frees
 *     device memory. Its only device memory of its own is the static
 *     scratch array of conv2d_bwd_weight_noalloc (one per GPU, loaded with
 *     the library), and no call reads what an earlier call left there, so it
 *     keeps no device state between calls. Its host state is two small
 *     records: the optimizer's per-workspace record of which layers have
 *     norms and which are applied in the current step (lars_adam_norms /
 *     lars_adam_apply, under a mutex), and the one-shot profiling events of
 *     fg_profile_next_launch (per host thread).
 *   - GPU work is enqueued on `stream` (0 = the null stream) and the call
 *     returns without synchronising; results are valid once the caller has
 *     synchronised the stream. Device faults surface at that synchronisation.
 *   - Arguments are validated on the host before any HIP call:
 *       FG_EINVAL        null pointer, non-positive size, empty output,
 *                        gate missing for FG_EPI_GATE, an output aliasing an
 *                        input, a gate overlapping the output other than
 *                        being the output itself, an unknown enum value;
 *       FG_EUNSUPPORTED  a valid shape outside what the kernels implement
 *                        (listed per call);
 *       FG_EWORKSPACE    ws_bytes below fg_conv_workspace_bytes();
 *       FG_ELAUNCH       the HIP runtime rejected a launch.
 *     No exception crosses the interface. On any error nothing is launched
 *     (FG_ELAUNCH: kernels launched before the failing one stay queued).
 *   - Results are bit-reproducible for a fixed device, shape and input:
 *     every sum is evaluated in a fixed order (no floating-point atomics).
 *   - Tensor sizes must stay below 2^31 elements per tensor.
 */
#ifndef FCNGRAD_H
#define FCNGRAD_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    FG_OK = 0,
    FG_EINVAL = 1,
    FG_EUNSUPPORTED = 2,
    FG_EWORKSPACE = 3,
    FG_ELAUNCH = 4
} fg_status;

/* Epilogue fused into the convolution's output.
 *   FG_EPI_NONE  out = fp16(acc)
 *   FG_EPI_RELU  out = fp16(acc > 0 ? acc : +0)          (forward ReLU)
 *   FG_EPI_ACC   out = fp16(out + acc): the result is added to what the
 *                output holds (gradient contributions summed in place; the
 *                staged store rounds acc to fp16 before the addition). Not
 *                for the K = 1 head (FG_EUNSUPPORTED).
 *   FG_EPI_GATE  out = fp16(gate > 0 ? acc : +0)         (ReLU backward;
 *                gate = the forward ReLU output at the same index, an fp16
 *                tensor with the output's shape)
 * acc is the fp32 accumulator; fp16() rounds to nearest-even with overflow
 * to +-infinity (no saturation) and keeps subnormals. */
typedef enum {
    FG_EPI_NONE = 0, FG_EPI_RELU = 1, FG_EPI_GATE = 2, FG_EPI_ACC = 3
} fg_epilogue;

/* Shape of a convolution, always described by its forward direction:
 *   n, h, w, c   the input image (NHWC); for the transposed convolution, its
 *                (smaller) input with c = C_in;
 *   k            output channels (transposed convolution: C_out);
 *   r, s         kernel height and width;
 *   stride_*, pad_*  stride and symmetric zero padding. */
typedef struct {
    int32_t n, h, w, c;
    int32_t k, r, s;
    int32_t stride_h, stride_w, pad_h, pad_w;
    /* Pixel strides, in elements, of the x-shaped tensors (x, dx) and the
     * y-shaped ones (y, dy); 0 means dense (c, resp. k). A stride other
     * than dense is honoured for
     *   - the pass's output (y of conv2d_fwd and conv_transpose2d_fwd, dx
     *     of conv2d_bwd_data), so that a pass can write into a channel
     *     slice of a wider buffer;
     *   - x where conv2d_fwd and conv2d_bwd_weight read it, so that a pass
     *     can read a channel slice (a dense block's layer reads the
     *     channels before those it writes, in the same buffer).
     * The pointer then addresses the slice's first channel. The stride
     * must be >= the channel count and a multiple of 8, the pointer 16-byte
     * aligned, and pixels * stride below 2^31 (else FG_EUNSUPPORTED; below
     * the channel count, FG_EINVAL). A gate is laid out like the output.
     * An input and an output at one stride whose channel ranges are
     * disjoint within each pixel do not overlap. Other tensors, and the
     * K = 1 head's, are dense (FG_EUNSUPPORTED otherwise). */
    int32_t x_ld, y_ld;
} fg_conv_desc;

/* One member of a gradient group: `ptr` is a device address (fp16 dW for
 * pack, fp32 destination for unpack), `numel` its element count and
 * `offset` the element offset of its first element inside the group. */
typedef struct {
    uint64_t ptr;
    uint64_t numel;
    uint64_t offset;
} fg_segment;

enum { FG_OP_FWD = 0, FG_OP_BWD_DATA = 1, FG_OP_BWD_WEIGHT = 2, FG_OP_CONVT = 3 };

/* Maximum number of members in one pack / unpack call. */
#define FG_MAX_SEGMENTS 64

/* ---- convolution passes (Section 5.2, OPS_conv and the factor 3) -------- */

/* Forward convolution: y[n,p,q,k] = epi(sum_{r,s,c} x~[n, p*sh-ph+r,
 * q*sw-pw+s, c] * w[k,r,s,c]), x~ = x extended by zeros outside the image.
 * x: n*h*w*c fp16; w_krsc: k*r*s*c fp16; y: n*P*Q*k fp16 (written);
 * gate: n*P*Q*k fp16 for FG_EPI_GATE, else ignored (may be NULL).
 * ws: device workspace of at least fg_conv_workspace_bytes(d, FG_OP_FWD)
 * bytes (may be NULL when that is 0); its contents are scratch.
 * FG_EUNSUPPORTED unless c % 8 == 0 and either k % 8 == 0, or k == 1 with a
 * 1x1 stride-1 unpadded kernel. Kernel sizes up to 4x4 (at most 16 taps). */
fg_status conv2d_fwd(const fg_conv_desc *d, const uint16_t *x,
                     const uint16_t *w_krsc, uint16_t *y, fg_epilogue epi,
                     const uint16_t *gate, void *ws, size_t ws_bytes,
                     hipStream_t stream);

/* Input gradient (adjoint of conv2d_fwd with respect to x):
 * dx[n,h,w,c] = epi(sum over k and the taps (r,s) with h + ph - r = p*sh and
 * w + pw - s = q*sw for some output position (p,q), of dy[n,p,q,k] *
 * w[k,r,s,c]); zero where no term lands. dy: n*P*Q*k; dx: n*h*w*c written;
 * gate: n*h*w*c for FG_EPI_GATE. Strided cases are evaluated per output
 * phase (h mod sh, w mod sw) over the taps that reach it only.
 * FG_EUNSUPPORTED unless c % 8 == 0 and (k % 8 == 0, or k == 1 with a 1x1
 * stride-1 unpadded kernel). */
fg_status conv2d_bwd_data(const fg_conv_desc *d, const uint16_t *dy,
                          const uint16_t *w_krsc, uint16_t *dx,
                          fg_epilogue epi, const uint16_t *gate, void *ws,
                          size_t ws_bytes, hipStream_t stream);

/* Kernel gradient: dw[k,r,s,c] = sum_{n,p,q} dy[n,p,q,k] *
 * x~[n, p*sh-ph+r, q*sw-pw+s, c], accumulated in fp32 and rounded once to
 * fp16. x: n*h*w*c; dy: n*P*Q*k; dw_krsc: k*r*s*c written. The reduction
 * over n*P*Q may be split across workgroups (fp32 partials in ws, summed in
 * a fixed order). FG_EUNSUPPORTED unless c % 8 == 0 and (k % 8 == 0, or
 * k == 1 with a 1x1 stride-1 unpadded kernel). */
fg_status conv2d_bwd_weight(const fg_conv_desc *d, const uint16_t *x,
                            const uint16_t *dy, uint16_t *dw_krsc, void *ws,
                            size_t ws_bytes, hipStream_t stream);

/* Kernel gradient straight into a gradient group (zero-copy fusion buffer,
 * Section 4.2 Grouping, with the non-finite check of Section 6.2 loss
 * scaling fused into its store). Computes exactly what conv2d_bwd_weight
 * computes, same arguments and errors, and in addition sets
 * *found_nonfinite (device int32) to 1 if any fp16 element written to
 * dw_krsc is +-inf or NaN; it never clears it. dw_krsc may point into a
 * group buffer at a member's element offset (16-byte aligned, as
 * grad_group_plan's 256-byte alignment guarantees), which makes that
 * member's grad_group_pack unnecessary. found_nonfinite must not be null
 * (FG_EINVAL) and must not overlap x, dy, dw_krsc or ws. */
fg_status conv2d_bwd_weight_checked(const fg_conv_desc *d, const uint16_t *x,
                                    const uint16_t *dy, uint16_t *dw_krsc,
                                    int32_t *found_nonfinite, void *ws,
                                    size_t ws_bytes, hipStream_t stream);

/* Size of the library's static scratch used by conv2d_bwd_weight_noalloc:
 * one copy per GPU, held until the process ends. */
#define FG_NOALLOC_SCRATCH_BYTES (64u << 20)

/* Kernel gradient without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc). Computes what conv2d_bwd_weight computes
 * (same validation and errors, ws aside); the fp32 split partials go to a
 * static FG_NOALLOC_SCRATCH_BYTES (64 MiB) device array of the library instead
 * of a caller workspace, and the split count is limited so that they fit: the
 * result is bit-identical to conv2d_bwd_weight whenever that call's workspace
 * (fg_conv_workspace_bytes) is at most FG_NOALLOC_SCRATCH_BYTES, and otherwise
 * the same sum in fewer, longer split ranges (a different fp32 order).
 * Nothing is allocated or freed (no hipMalloc, hipFree or allocating library
 * call); the first call on a device looks up that device's copy of the scratch
 * (FG_ELAUNCH if the runtime cannot). Every call on one GPU shares that GPU's
 * scratch: calls that overlap in time on one GPU (other streams, other host
 * threads) race and must be ordered by the caller. No part of the scratch needs
 * clearing between calls. FG_EWORKSPACE if a plan would need more scratch than
 * FG_NOALLOC_SCRATCH_BYTES (not reached by shapes the library accepts). */
fg_status conv2d_bwd_weight_noalloc(const fg_conv_desc *d, const uint16_t *x,
                                    const uint16_t *dy, uint16_t *dw_krsc,
                                    hipStream_t stream);

/* Transposed convolution (decoder upsampling):
 * y[n,o,u,k] = epi(sum over c and the taps (r,s) with o + ph - r = i*sh and
 * u + pw - s = j*sw for an input position (i,j), of x[n,i,j,c] *
 * w[c,r,s,k]). Output size (h-1)*sh - 2*ph + r by (w-1)*sw - 2*pw + s.
 * x: n*h*w*c (c = C_in); w_crsk: c*r*s*k; y written; gate shaped like y.
 * Its backward passes are conv2d_fwd (input gradient: dy convolved with
 * w_crsk read as a KRSC weight with K = C_in, C = C_out) and
 * conv2d_bwd_weight (x := dy, dy := x). FG_EUNSUPPORTED unless c % 8 == 0,
 * k % 8 == 0 and the kernel is 4x4 with stride 2 and padding 1. */
fg_status conv_transpose2d_fwd(const fg_conv_desc *d, const uint16_t *x,
                               const uint16_t *w_crsk, uint16_t *y,
                               fg_epilogue epi, const uint16_t *gate,
                               void *ws, size_t ws_bytes, hipStream_t stream);

/* ---- gradient path (Section 4.2 Grouping; Section 6.2 loss scaling) ----- */

/* Fusion-buffer copy-in: group[seg.offset + j] = src[j] (bit copy) for every
 * segment, and every element of [0, group_numel) not covered by a segment
 * is set to 0x0000. segs: host array of nseg (1..FG_MAX_SEGMENTS) fp16
 * sources, read during the call only; segments must lie inside the group
 * and must not overlap each other (FG_EINVAL). A segment may have no
 * elements (its ptr may then be NULL): it copies nothing, and its place is
 * zero-filled like any uncovered element. group: group_numel fp16. */
fg_status grad_group_pack(const fg_segment *segs, int32_t nseg,
                          uint16_t *group, uint64_t group_numel,
                          hipStream_t stream);

/* Loss-scale removal with overflow detection:
 * out_f32[j] = fp32(value(group[j]) * inv_scale), one nearest-even rounding
 * of the exact product, for j < numel; and *found_nonfinite is set to 1 if
 * any group[j] has an all-ones exponent field (+-inf or NaN). The flag is
 * only ever written with 1: the caller zeroes it before the step and may
 * share one flag between several calls. */
fg_status grad_unscale_check(const uint16_t *group, uint64_t numel,
                             float inv_scale, float *out_f32,
                             int32_t *found_nonfinite, hipStream_t stream);

/* Clears n device int32 non-finite flags (flags[0..n) = 0) with a kernel on
 * `stream` (no memset node, so the call may sit in a captured graph). The
 * flags grad_unscale_check and conv2d_bwd_weight_checked raise are only
 * ever set, so a step clears them before its first check. FG_EINVAL for a
 * null pointer or n < 1. */
fg_status grad_flags_clear(int32_t *flags, int32_t n, hipStream_t stream);

/* Fusion-buffer copy-out: dst[j] = group_f32[seg.offset + j] (bit copy) for
 * every segment; seg.ptr is the fp32 destination. Same segment rules as
 * grad_group_pack (group_numel bounds the offsets); the destinations of
 * non-empty segments must not overlap each other (FG_EINVAL), and a segment
 * with no elements writes nothing. */
fg_status grad_group_unpack(const float *group_f32, uint64_t group_numel,
                            const fg_segment *segs, int32_t nseg,
                            hipStream_t stream);

/* ---- network glue (Section 6.2, Model Implementation) -------------------- */

/* Gradient of the loss-scaled mean squared error at the network output:
 * dy[j] = fp16(scale * (y[j] - t[j])), evaluated in fp64 and rounded once
 * to fp16 (nearest-even, overflow to infinity); for loss S * mean((y-t)^2)
 * over numel outputs the caller passes scale = 2*S/numel. y fp16, t fp32. */
fg_status l2_head_grad(const uint16_t *y, const float *t, uint64_t numel,
                       double scale, uint16_t *dy, hipStream_t stream);

/* Gradient through a ReLU where no convolution follows to fuse it into:
 * out[j] = act[j] > 0 ? dy[j] : +0 (bit copy of dy when passed). */
fg_status relu_backward(const uint16_t *dy, const uint16_t *act,
                        uint64_t numel, uint16_t *out, hipStream_t stream);

/* ---- host-only helpers (no device access) ------------------------------- */

/* Backoff loss scaling (Section 6.2, Model Implementation: the loss is
 * scaled before the gradient computation, adaptively). A step whose
 * gradients hold a non-finite value is not applied and halves the scale
 * (not below s_min), restarting the count of clean steps; after `interval`
 * clean steps in a row the scale doubles (not above s_max). Powers of two
 * keep scaling and unscaling exact. */
typedef struct {
    double scale;      /* the loss scale S of the next step */
    int32_t clean;     /* clean steps since the last change of S */
    int32_t interval;  /* clean steps before S doubles (>= 1) */
    double s_min, s_max;
} fg_loss_scale;

/* Records one step's outcome in *s (found_nonfinite: the step's flags, any
 * non-zero) and sets *applied to 1 if the step's update applies, else 0.
 * FG_EINVAL for null pointers, interval < 1, or a state outside
 * 0 < s_min <= scale <= s_max (nothing is changed then). */
fg_status fg_loss_scale_update(fg_loss_scale *s, int32_t found_nonfinite,
                               int32_t *applied);

/* Learning rate per applied step (Section 6.2: a linear warm-up of the rate
 * from base to about N times base for N ranks, then a staircase decay):
 * lr(k) = base + (peak - base) * k / warmup for k < warmup, else
 * peak * rate^floor((k - warmup) / every) (every = 0: no decay). k counts
 * applied updates from 0. FG_EINVAL for null pointers, k < 0, negative
 * base, peak, warmup or every, or a rate not in (0, +inf). */
typedef struct {
    double base, peak;
    int64_t warmup, every;
    double rate;
} fg_lr_schedule;

fg_status fg_lr_at(const fg_lr_schedule *s, int64_t k, double *lr);

/* Measurement: the sustained fp16 MFMA rate of this GPU, the on-chip
 * ceiling against which the convolutions' rates (Section 5.2, Sustained and
 * Peak) can be read beside the nominal peak. Launches `blocks` workgroups of
 * 4 waves; every wave runs `iters` iterations of 8 v_mfma_f32_32x32x16_f16
 * from registers only (4 accumulator chains, no memory traffic in the loop),
 * then each of its threads writes one float, the sum of its accumulators, to
 * out[blockIdx * 256 + thread] (device, blocks * 256 floats, owned by the
 * caller). Work: blocks * iters * 2^20 flops. Operands are hashed from the
 * thread, operand and element indices, about half zero: operands = 0 gives
 * random fp16 values in (-1, 1), which draw the power of real data;
 * operands = 1 gives integers in -2..2, whose sums stay exact in fp32.
 * FG_EINVAL for a null out, blocks or iters < 1, another operands value, or
 * blocks * iters above FG_MFMA_LOOP_MAX_WORK (about 0.1 s of work). */
#define FG_MFMA_LOOP_MAX_WORK (1LL << 28)
fg_status fg_mfma_loop(float *out, int32_t blocks, int32_t iters, int32_t operands,
                       hipStream_t stream);

/* Profiling: the next convolution call (conv2d_fwd, conv2d_bwd_data,
 * conv2d_bwd_weight[_checked], conv_transpose2d_fwd) made on this host
 * thread records `start` on its stream just before its main kernel and
 * `stop` just after it, so that the main kernel's duration can be read with
 * hipEventElapsedTime apart from a split reduction launched after it. The
 * events are then forgotten; calls that fail validation leave them armed.
 * Either may be null (disarms). The caller owns the events. */
fg_status fg_profile_next_launch(hipEvent_t start, hipEvent_t stop);

/* Workspace in bytes that the given pass needs for this shape (0 if none). */
size_t fg_conv_workspace_bytes(const fg_conv_desc *d, int op);

/* ---- optimizer (Section 6.2: layer-wise adaptive rates with Adam) ------ */

/* One layer for lars_adam_update: device addresses of its fp32 master
 * weights (w32, read and written), fp16 working weights (w16, written), fp32
 * Adam moments (m, v, read and written) and fp32 unscaled gradient (g, read);
 * numel elements each (1 .. 2^31 - 1). w32, m, v and g 16-byte aligned, w16
 * 8-byte aligned; no two arrays of the call may overlap. */
typedef struct {
    uint64_t w32, w16, m, v, g;
    uint64_t numel;
} fg_opt_tensor;

typedef struct {
    float lr, beta1, beta2, eps, weight_decay;
} fg_opt_params;

/* Workspace (bytes, device) the optimizer calls need for these layers (it
 * depends on the element counts only); 0 for a count outside
 * 1..FG_MAX_SEGMENTS or a numel outside 1..2^31 - 2. */
size_t fg_lars_adam_workspace_bytes(const fg_opt_tensor *t, int32_t ntensors);

/* Form of the gradient t[i].g of the optimizer calls: fp32 unscaled
 * (16-byte aligned), or fp16 loss-scaled (8-byte aligned, e.g. the layer's
 * slot in its gradient group buffer), read as fp16 * grad_inv_scale — the
 * fp32 value grad_unscale_check writes for it. */
enum { FG_GRAD_F32 = 0, FG_GRAD_F16_SCALED = 1 };

/* Layer-wise adaptive Adam step on fp32 master weights (Section 6.2: LARS
 * layer-wise rates with Adam, L2 weight decay). For each layer, with
 * t = *step_count + 1: g~ = g + weight_decay * w; m = beta1 m + (1-beta1) g~;
 * v = beta2 v + (1-beta2) g~^2; u = (m / (1-beta1^t)) / (sqrt(v /
 * (1-beta2^t)) + eps); tau = ||w|| / ||u|| over the layer (1 if either is
 * 0); w = w - lr * tau * u; w16 = nearest-even fp16 of the new w; then
 * *step_count = t. If any of the nflags device int32 found_nonfinite flags
 * (the unscale checks of the step's gradient groups) is non-zero, the step
 * is skipped on the device: nothing is written and *step_count is kept.
 * fp32 arithmetic; per-layer norms summed in a fixed order (the result is
 * deterministic). The square root and the quotient of u are the hardware
 * ones (a few ulps). t: host array of ntensors (1..FG_MAX_SEGMENTS) layers
 * with fp32 gradients, read during the call only. FG_EINVAL for null or
 * misaligned pointers, overlapping arrays, params outside lr >= 0,
 * 0 <= beta < 1, eps >= 0, weight_decay >= 0, nflags > 0 with null flags,
 * or flags overlapping ws, the step count or an array the update writes;
 * FG_EWORKSPACE if ws_bytes is short or ws is not 16-byte aligned.
 * Same as lars_adam_norms over all layers followed by lars_adam_apply. */
fg_status lars_adam_update(const fg_opt_tensor *t, int32_t ntensors,
                           const fg_opt_params *p,
                           const int32_t *found_nonfinite, int32_t nflags,
                           int32_t *step_count, void *ws, size_t ws_bytes,
                           hipStream_t stream);

/* The update of lars_adam_update in parts, so that the part that reads each
 * layer's gradient can run as soon as that gradient exists (e.g. per
 * gradient group, beside the rest of the backward pass), and each layer's
 * writes just before that layer's weights are next read (e.g. the next
 * forward pass, layer by layer).
 * lars_adam_norms reads layers [first, first + count) of the table t
 * (weights, moments, gradient; nothing is written but ws) and stores their
 * partial sums of u^2 and w^2 in ws; t = *step_count + 1 as in
 * lars_adam_update. lars_adam_apply, once norms calls have covered every
 * layer, writes m, v, w and the fp16 copy of layers [first, first + count)
 * as lars_adam_update does, or nothing if a flag is set; the first apply
 * call of a step also forms every layer's tau and advances *step_count (or
 * leaves it if a flag is set). Between the first norms call and the apply
 * call that completes the table, the caller passes the same table, params
 * (lr aside), gradient form, grad_inv_scale, step_count and ws, changes
 * none of the layer arrays, and orders every apply after every norms call
 * and later applies after the first on the device (same stream, or
 * events). Validation as lars_adam_update, with the gradient form
 * (FG_GRAD_*), for fp16 gradients a finite grad_inv_scale > 0, and a range
 * inside the table. Tracked on the host per workspace address, before any
 * launch: lars_adam_apply returns FG_EINVAL unless norms calls with these
 * arguments have covered every layer since the last completed apply and
 * its range holds no layer already applied in this step; lars_adam_norms
 * returns FG_EINVAL while the apply of a step is incomplete. A
 * lars_adam_update on ws clears the record. */
fg_status lars_adam_norms(const fg_opt_tensor *t, int32_t ntensors, int32_t first,
                          int32_t count, const fg_opt_params *p, int32_t grad_format,
                          float grad_inv_scale, const int32_t *step_count, void *ws,
                          size_t ws_bytes, hipStream_t stream);
fg_status lars_adam_apply(const fg_opt_tensor *t, int32_t ntensors, int32_t first,
                          int32_t count, const fg_opt_params *p, int32_t grad_format,
                          float grad_inv_scale, const int32_t *found_nonfinite,
                          int32_t nflags, int32_t *step_count, void *ws,
                          size_t ws_bytes, hipStream_t stream);

/* ---- FC-DenseNet variant (Section 6.2, Neural Network Architecture and
 * Model Implementation) ---------------------------------------------------- */

/* Gradient of the loss-scaled mean Huber loss (Section 6.2, the loss
 * equation, with cutoff delta): dy[j] = fp16(scale * clamp(y[j] - t[j],
 * -delta, delta)), evaluated in fp64 and rounded once (nearest-even,
 * overflow to infinity). For the loss S * mean(huber_delta(y - t)) over
 * numel outputs, where huber_delta(d) = d^2/2 for |d| <= delta and
 * delta (|d| - delta/2) beyond, the caller passes scale = S/numel. y fp16,
 * t fp32, dy fp16; numel 1..2^31-1. FG_EINVAL for null pointers, delta not
 * > 0 (+inf is allowed and gives scale * (y - t)), a non-finite scale, or dy
 * overlapping y or t. */
fg_status huber_head_grad(const uint16_t *y, const float *t, uint64_t numel,
                          double scale, double delta, uint16_t *dy,
                          hipStream_t stream);

/* 2x2 average pooling with stride 2 (Section 6.2: average pooling in place
 * of max pooling). x: N x H x W x C fp16 (NHWC), H and W even; y: N x H/2 x
 * W/2 x C, the mean of the four inputs computed exactly and rounded once.
 * FG_EINVAL for null or overlapping buffers or a non-positive size;
 * FG_EUNSUPPORTED for odd H or W, C not a multiple of 8, 2^31 or more
 * elements, or a pointer not 16-byte aligned. */
fg_status avg_pool2d_fwd(const uint16_t *x, int32_t n, int32_t h, int32_t w, int32_t c,
                         uint16_t *y, hipStream_t stream);

/* Gradient of avg_pool2d_fwd: dx[n, 2p+i, 2q+j, c] = fp16(dy[n, p, q, c] / 4),
 * or +0 where gate (N x H x W x C fp16, e.g. the ReLU output that was
 * pooled; may be null) is <= 0. n, h, w, c are the forward input's sizes.
 * Same checks as the forward; dx may not overlap dy or gate. */
fg_status avg_pool2d_bwd(const uint16_t *dy, const uint16_t *gate, int32_t n, int32_t h,
                         int32_t w, int32_t c, uint16_t *dx, hipStream_t stream);

/* Channel slice copy between NHWC buffers with their own pixel strides
 * (Section 6.2: dense blocks concatenate their layers' outputs along the
 * channels, growth rate 256). For npix pixels p and channels k < nch:
 * v = src[p*src_ld + k], or +0 where gate[p*gate_ld + k] <= 0 (gate may be
 * null); dst[p*dst_ld + k] = v, or fp16(dst[p*dst_ld + k] + v) (exact sum,
 * one rounding) when accumulate is non-zero. A slice at channel offset o is
 * addressed by offsetting the pointer by o. The concatenation of a dense
 * block is a copy of each piece into its slice; backward, a slice's
 * gradient is read out (gated by the piece's ReLU output) and a layer's
 * input gradient is accumulated into the slices it read. FG_EINVAL for a
 * null src or dst, non-positive sizes or strides, nch above a stride, or
 * dst's span ((npix-1)*dst_ld + nch elements) overlapping src's or gate's;
 * FG_EUNSUPPORTED for nch or a stride not a multiple of 8, a pointer not
 * 16-byte aligned, or npix times a stride of 2^31 or more. */
fg_status channel_slice_copy(const uint16_t *src, int32_t src_ld, const uint16_t *gate,
                             int32_t gate_ld, uint16_t *dst, int32_t dst_ld, int64_t npix,
                             int32_t nch, int32_t accumulate, hipStream_t stream);

/* Output spatial size: transpose = 0 gives the forward P, Q; 1 gives the
 * transposed convolution's output size. FG_EINVAL if it is not positive. */
fg_status fg_conv_out_dims(const fg_conv_desc *d, int transpose, int32_t *p,
                           int32_t *q);

/* Group planner (Section 4.2, Grouping; Figure grouping). Tensors are given
 * in backward-completion order (numel[i] elements of elem_bytes each). A
 * tensor joins the open group at the next multiple of align_bytes unless
 * its end would pass cap_bytes, in which case the open group is closed
 * first; a tensor larger than the cap forms a group of its own. Outputs:
 * group_of[i], offset_of[i] (elements), *ngroups and group_numel[g] (the
 * end of the group's last member; arrays sized ntensors). */
fg_status grad_group_plan(const uint64_t *numel, int32_t ntensors,
                          uint64_t cap_bytes, uint32_t align_bytes,
                          uint32_t elem_bytes, int32_t *group_of,
                          uint64_t *offset_of, int32_t *ngroups,
                          uint64_t *group_numel);

/* Name of the main GPU kernel the given pass launches for this shape (a
 * static string; "" for an invalid or unsupported shape). Lets a profiler
 * or benchmark group launches the way a kernel trace does. */
const char *fg_conv_kernel_name(const fg_conv_desc *d, int op);

/* Human-readable name of a status code (static string). */
const char *fg_status_string(fg_status s);

#ifdef __cplusplus
}
#endif
#endif /* FCNGRAD_H */
