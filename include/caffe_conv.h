/*
 * caffe_conv.h -- C ABI of the MI355X (gfx950) convolution-layer library
 * (libcaffe_conv.so).
 *
 * The operation is the convolution layer of Caffe (Jia et al., "Caffe:
 * Convolutional Architecture for Fast Feature Embedding", 2014).  Sec. 3.1
 * fixes the data: 4-D blobs (here N x C x H x W, row-major, "NCHW").
 * Sec. 3.2 fixes the roles: the forward pass maps the input blob to the
 * output blob; the backward pass maps the gradient w.r.t. the output to the
 * gradients w.r.t. the parameters (weights, bias) and w.r.t. the input.
 * Sec. 3.2 also lists rectified-linear units, which this library can fuse
 * into the convolution.  The paper gives no formula; the library computes the
 * textbook strided, zero-padded, grouped 2-D cross-correlation:
 *
 *   Ho = floor((H + 2 pad_h - kernel_h) / stride_h) + 1   (Wo likewise)
 *   Cg = C / group, Kg = K / group, output channel k belongs to group t = k / Kg
 *   Z[n,k,i,j] = bias[k] + sum_{c<Cg, u<kh, v<kw}
 *                weight[k,c,u,v] * bottom[n, t*Cg + c, i*sh - ph + u, j*sw - pw + v]
 *                (bottom reads as 0 outside the image, no kernel flip)
 *   top = relu ? max(Z, 0) : Z
 *
 * and, with D = relu ? top_diff * [top > 0] : top_diff,
 *
 *   bias_diff[k]       = sum_{n,i,j} D[n,k,i,j]
 *   weight_diff[k,c,u,v] = sum_{n,i,j} D[n,k,i,j] * bottom[n, t*Cg + c, i*sh - ph + u, j*sw - pw + v]
 *   bottom_diff        = the adjoint of the forward map applied to D.
 *
 * Layouts.  bottom / bottom_diff: N x C x H x W.  weight / weight_diff:
 * K x Cg x kernel_h x kernel_w.  bias / bias_diff: K.  top / top_diff:
 * N x K x Ho x Wo.  All dense, row-major, no strides.
 *
 * Types.  `desc->dtype` selects the operand type of `bottom` and `weight`:
 * CAFFE_F32 (float) or CAFFE_BF16 (bfloat16 stored as uint16_t; the caller
 * rounds to nearest-even).  CAFFE_BF16_F32_BOTTOM is CAFFE_BF16 with a float
 * `bottom` that the library rounds to bfloat16 (nearest-even) as it copies it
 * into its workspace, so the products, results and gradients are those of
 * CAFFE_BF16 on the rounded bottom (CAFFE_BACKWARD_MASK_BOTTOM_DIFF keeps
 * the gradient where the rounded value is > 0): it saves the caller a
 * separate rounding pass over the layer's input.  Everything else (bias, top,
 * top_diff, every gradient) is float in all modes, and every product is
 * accumulated in float.  In both bf16 modes `top_diff` (after the ReLU mask)
 * is rounded to bfloat16 (nearest-even) before it enters a product;
 * bias_diff sums the unrounded float values.
 *
 * Memory and ownership.  Every tensor pointer is a device pointer (HIP
 * device memory of the current device), allocated and owned by the caller,
 * 16-byte aligned.  The library never allocates, frees or retains caller
 * memory.  Scratch space comes from the caller as `workspace` / `ws_bytes`
 * (device memory, 256-byte aligned); query the size with
 * caffe_conv_workspace_size().  No tensor may exceed 2^31 - 1 bytes.
 *
 * Execution.  Every compute call only validates its arguments on the host
 * and enqueues kernels on `stream` (a hipStream_t; NULL = the default
 * stream), then returns: the results are ready when the stream reaches that
 * point.  Device faults therefore surface at the caller's next
 * synchronisation.  Calls on different streams that share no output or
 * workspace memory may run concurrently; the library's only global state is
 * one auxiliary stream per device, created on first use by
 * caffe_conv_backward.  Results are bitwise reproducible run to run for the
 * same arguments (no atomics; every sum has a fixed order).
 *
 * Errors.  Every call returns CAFFE_OK (0) or a negative caffe_status.  A
 * call that fails its argument checks (every code but CAFFE_ERR_HIP) has
 * enqueued nothing.  CAFFE_ERR_HIP means the HIP runtime refused a launch or
 * a stream operation part-way through: the kernels the call had already
 * enqueued on `stream` stay enqueued (the call's outputs are then undefined),
 * and work it had forked to the auxiliary stream has finished before the
 * call returns.  caffe_status_string() names a code; caffe_last_error()
 * returns a thread-local message describing the last failure on the calling
 * thread.
 *
 * Tuning.  Tile shapes, split counts and kernel variants are chosen from the
 * descriptor alone.  Environment variables named CAFFE_CONV_*, CAFFE_FC_*,
 * CAFFE_BF16_* and CAFFE_BACKWARD_FORK override those choices for profiling
 * and tests, and are read only while CAFFE_PROFILE_OVERRIDES=1 is set.
 */
#ifndef CAFFE_CONV_H
#define CAFFE_CONV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum caffe_status {
    CAFFE_OK = 0,
    CAFFE_ERR_INVALID_ARG = -1, /* bad shape, NULL required pointer, bad flag      */
    CAFFE_ERR_ALIGN = -2,       /* pointer not 16-byte (workspace: 256-byte) aligned */
    CAFFE_ERR_WORKSPACE = -3,   /* ws_bytes smaller than caffe_conv_workspace_size   */
    CAFFE_ERR_UNSUPPORTED = -4, /* unknown dtype, or a tensor of 2^31 bytes or more  */
    CAFFE_ERR_HIP = -5          /* the HIP runtime refused a launch                  */
} caffe_status;

typedef enum caffe_dtype {
    CAFFE_F32 = 0,
    CAFFE_BF16 = 1,
    CAFFE_BF16_F32_BOTTOM = 2 /* bf16 weight, float bottom rounded by the library */
} caffe_dtype;

/* Layer geometry: the parameters Caffe's convolution layer is defined by. */
typedef struct caffe_conv_desc {
    int32_t N, C, H, W;           /* bottom blob; N may be 0 (empty batch)        */
    int32_t K;                    /* number of output channels (filters)          */
    int32_t kernel_h, kernel_w;   /* >= 1                                         */
    int32_t stride_h, stride_w;   /* >= 1                                         */
    int32_t pad_h, pad_w;         /* >= 0, zero padding on both sides             */
    int32_t group;                /* >= 1, divides C and K; contiguous channel slices */
    int32_t relu;                 /* 0 or 1: fuse max(., 0) after the bias        */
    int32_t dtype;                /* caffe_dtype of bottom and weight             */
} caffe_conv_desc;

enum caffe_conv_pass {
    CAFFE_PASS_FORWARD = 0,
    CAFFE_PASS_BACKWARD_DATA = 1,
    CAFFE_PASS_BACKWARD_WEIGHTS = 2,
    CAFFE_PASS_BACKWARD = 3, /* caffe_conv_backward: data and weights together */
    CAFFE_PASS_BACKWARD_POOL_LRN = 4 /* caffe_conv_backward_pool_lrn (caffe_layers.h) */
};

/* Output spatial size (formula above).  Host-only; never touches a GPU.
 * Returns CAFFE_ERR_INVALID_ARG for an invalid descriptor. */
int caffe_conv_out_shape(const caffe_conv_desc* desc, int32_t* Ho, int32_t* Wo);

/* Bytes of device workspace that `pass` (a caffe_conv_pass) needs for this
 * descriptor; 0 is a valid answer.  Host-only. */
int caffe_conv_workspace_size(const caffe_conv_desc* desc, int32_t pass, size_t* bytes);

/* The same query returning the size: SIZE_MAX for an invalid descriptor or
 * pass (caffe_last_error() then says why).  Host-only. */
size_t caffe_conv_workspace_bytes(const caffe_conv_desc* desc, int32_t pass);

/* Forward pass (Sec. 3.2): top = [relu](weight (*) bottom + bias).
 * bias may be NULL (no bias).  top is overwritten. */
int caffe_conv_forward(const caffe_conv_desc* desc, const void* bottom, const void* weight,
                       const float* bias, float* top, void* workspace, size_t ws_bytes,
                       void* stream);

/* Flags of caffe_conv_forward_ex. */
enum caffe_forward_flags {
    /* bf16 modes: the workspace already holds bottom's staged bf16 copy,
     * written by caffe_pool_lrn_forward_into (caffe_layers.h) for this
     * descriptor and workspace; the call does not stage bottom again (bottom
     * may be NULL) and the later backward's CAFFE_BACKWARD_BOTTOM_STAGED
     * reads that copy.  CAFFE_ERR_INVALID_ARG in CAFFE_F32 mode. */
    CAFFE_FORWARD_BOTTOM_STAGED = 1
};

/* caffe_conv_forward with caffe_forward_flags. */
int caffe_conv_forward_ex(const caffe_conv_desc* desc, const void* bottom, const void* weight,
                          const float* bias, float* top, void* workspace, size_t ws_bytes,
                          int32_t flags, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * caffe_conv_forward with its workspace taken from a static device array the
 * library owns, CAFFE_CONV_NOALLOC_SCRATCH_BYTES per device (each GPU the
 * library runs on keeps its copy until the process ends).  The call
 * allocates nothing; the caller still provides bottom, weight, bias and top.
 * Returns CAFFE_ERR_WORKSPACE when the forward pass needs more workspace
 * than that (caffe_conv_workspace_size with CAFFE_PASS_FORWARD tells in
 * advance), e.g. bf16 operands at CaffeNet conv1's size, whose staged input
 * alone is larger.  The first call on a device looks up the array's address
 * (a one-time set-up; nothing is allocated).  Every call on one device uses
 * the same array, and nothing in it needs to start at zero: calls that may
 * overlap in time on one device (different streams, or several host threads)
 * race on it, so the caller serialises them. */
#define CAFFE_CONV_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
int caffe_conv_forward_noalloc(const caffe_conv_desc* desc, const void* bottom,
                               const void* weight, const float* bias, float* top, void* stream);

/* Backward pass w.r.t. the input (Sec. 3.2): bottom_diff = adjoint(D).
 * top is the forward output and is required iff desc->relu; it is read only
 * for the mask [top > 0].  bottom_diff is overwritten. */
int caffe_conv_backward_data(const caffe_conv_desc* desc, const float* top_diff, const float* top,
                             const void* weight, float* bottom_diff, void* workspace,
                             size_t ws_bytes, void* stream);

/* Backward pass w.r.t. the parameters (Sec. 3.2): weight_diff and (if not
 * NULL) bias_diff.  accumulate = 0 overwrites them, 1 adds to them.  top is
 * required iff desc->relu. */
int caffe_conv_backward_weights(const caffe_conv_desc* desc, const float* top_diff,
                                const float* top, const void* bottom, float* weight_diff,
                                float* bias_diff, int32_t accumulate, void* workspace,
                                size_t ws_bytes, void* stream);

/* Flags of caffe_conv_backward: they let a network fold the backward pass of
 * the ReLUs around a layer into the neighbouring layers' kernels instead of
 * running it as a pass of its own. */
enum caffe_backward_flags {
    /* top_diff is already zero wherever top <= 0: the fused ReLU's backward
     * was applied by whoever produced top_diff.  top is then not read. */
    CAFFE_BACKWARD_TOP_DIFF_MASKED = 1,
    /* bottom_diff is stored multiplied by [bottom > 0]: the backward pass of
     * a ReLU whose output is this layer's bottom, fused into the data
     * gradient.  Needs bottom (in CAFFE_BF16 mode the mask is taken from
     * the bf16 bottom). */
    CAFFE_BACKWARD_MASK_BOTTOM_DIFF = 2,
    /* CAFFE_BF16 mode: the workspace still holds the staged copy of bottom
     * written by the last caffe_conv_forward call with the same descriptor,
     * bottom and workspace, and none of them has changed since (the
     * training-step order: forward, then backward on a workspace of its
     * own).  The weight gradient then reads that copy instead of staging
     * bottom again; the staged copy sits at the start of both passes'
     * workspaces.  No effect in CAFFE_F32 mode, which stages nothing; a
     * workspace that does not hold the forward's copy gives a wrong
     * weight gradient. */
    CAFFE_BACKWARD_BOTTOM_STAGED = 4,
    /* bf16 modes: the workspace holds this layer's staged top gradient and
     * its bias-gradient partial sums, written by the layer above's
     * caffe_conv_backward_into (which named this descriptor and workspace
     * as `below`); top_diff is not read (it may be NULL) and counts as
     * masked.  CAFFE_ERR_INVALID_ARG in CAFFE_F32 mode. */
    CAFFE_BACKWARD_TOP_STAGED = 16,
    /* caffe_conv_backward_pool_lrn(_ex) (caffe_layers.h) only: pool_mask
     * holds one byte per pooled value, as caffe_pool_lrn_forward writes it
     * with CAFFE_POOL_MASK_OFFSETS. */
    CAFFE_BACKWARD_POOL_MASK_OFFSETS = 32
};

/* The whole backward pass of the layer in one call: the ReLU mask is applied
 * once and shared by both gradients.  Any of bottom_diff, weight_diff,
 * bias_diff may be NULL to skip it; bottom is required iff weight_diff is
 * given or flags has CAFFE_BACKWARD_MASK_BOTTOM_DIFF, weight iff bottom_diff
 * is given.  accumulate applies to weight_diff and bias_diff only; flags is a
 * set of caffe_backward_flags.  In CAFFE_BF16 mode with both bottom_diff and
 * weight_diff, the weight gradient runs on the device's auxiliary stream
 * (default priority), which waits for `stream` after the top gradient is
 * staged and which `stream` waits for before the call returns: the results
 * are ordered on `stream` as always.  Not while `stream` is being captured
 * into a graph, and not with CAFFE_BACKWARD_FORK=0 (read only while
 * CAFFE_PROFILE_OVERRIDES=1). */
int caffe_conv_backward(const caffe_conv_desc* desc, const float* top_diff, const float* top,
                        const void* bottom, const void* weight, float* bottom_diff,
                        float* weight_diff, float* bias_diff, int32_t accumulate, int32_t flags,
                        void* workspace, size_t ws_bytes, void* stream);

/* caffe_conv_backward with the weight-side outputs (weight_diff and
 * bias_diff) ordered on weight_stream instead of `stream` (the same call
 * when the two are equal).  weight_stream first waits for all work enqueued
 * on `stream` before the call, then, in the bf16 modes, for the top-gradient
 * staging the call enqueues there, and takes the weight and bias gradients
 * while `stream` goes on with the data gradient (bottom_diff, ordered on
 * `stream`); nothing joins the two streams, so a network can run one
 * layer's weight gradient beside the next layers' data gradients and glue.
 * In CAFFE_F32 mode both passes share the workspace's partial sums and run
 * on `stream`, which weight_stream then waits for.  The workspace stays in
 * use until both streams have passed the call's work; the caller joins the
 * streams before reusing it or reading weight_diff on `stream`.  The
 * default-priority stream rule of the backward's auxiliary stream applies
 * to weight_stream as well. */
int caffe_conv_backward_ex(const caffe_conv_desc* desc, const float* top_diff, const float* top,
                           const void* bottom, const void* weight, float* bottom_diff,
                           float* weight_diff, float* bias_diff, int32_t accumulate,
                           int32_t flags, void* workspace, size_t ws_bytes, void* stream,
                           void* weight_stream);

/* caffe_conv_backward_ex whose data gradient is not stored as a float
 * bottom_diff but written, rounded to bf16 (nearest even), as the staged top
 * gradient of the convolution `below` -- the layer whose top is this layer's
 * bottom -- in below's backward workspace (below_workspace, at least
 * caffe_conv_workspace_size(below, CAFFE_PASS_BACKWARD) bytes), together with
 * the partial sums below's bias gradient adds up, and with the zero border
 * below's data gradient gathers from.  With CAFFE_BACKWARD_MASK_BOTTOM_DIFF
 * the values are masked first, as bottom_diff would be.  below's backward
 * then takes CAFFE_BACKWARD_TOP_STAGED (on a stream ordered after `stream`)
 * and reads no float top gradient: the pass that would write, read back and
 * stage it is gone.  Requirements (else CAFFE_ERR_UNSUPPORTED): bf16 modes
 * for both layers, stride 1 with the data gradient's grid the image itself,
 * a multiple of 4 channels per group here and no channel padding in below's
 * staging (a multiple of 8 channels per group); below's N, K, Ho, Wo must be
 * this layer's N, C, H, W (CAFFE_ERR_INVALID_ARG). */
/* 1 when caffe_conv_backward_into can stage desc's data gradient for
 * `below` (the requirements above), else 0 (also for an invalid descriptor;
 * caffe_last_error() then says why).  Host-only. */
int caffe_conv_stage_below_supported(const caffe_conv_desc* desc, const caffe_conv_desc* below);

int caffe_conv_backward_into(const caffe_conv_desc* desc, const float* top_diff, const float* top,
                             const void* bottom, const void* weight, float* weight_diff,
                             float* bias_diff, int32_t accumulate, int32_t flags,
                             void* workspace, size_t ws_bytes, const caffe_conv_desc* below,
                             void* below_workspace, size_t below_ws_bytes, void* stream,
                             void* weight_stream);

/* Static name of a status code ("CAFFE_OK", ...). */
const char* caffe_status_string(int32_t status);

/* The same name under the convolution layer's prefix. */
const char* caffe_conv_status_string(int32_t status);

/* Thread-local text of the last error raised on this thread ("" if none). */
const char* caffe_last_error(void);

/* Library version, major * 10000 + minor * 100 + patch. */
int32_t caffe_version(void);

#ifdef __cplusplus
}
#endif

#endif /* CAFFE_CONV_H */
