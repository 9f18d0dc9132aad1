/*
 * caffe_layers.h -- C ABI of the glue layers that sit between CaffeNet's
 * convolutions, in the same library as caffe_conv.h (libcaffe_conv.so).
 *
 * Both layers are in the paper's list of Caffe layer types (Sec. 3.2:
 * pooling, local response normalisation), with the same forward/backward
 * roles as the convolution layer.  The paper gives no formulas; the library
 * computes:
 *
 * Max pooling: Ho = floor((H + 2 pad_h - kernel_h) / stride_h) + 1 (Wo
 * likewise); top[n,c,i,j] = max over rows i*sh - ph .. i*sh - ph + kh - 1 and
 * the matching columns, clipped to the image.  Ties go to the first maximum
 * in row-major window order.  `mask` (int32, N x C x Ho x Wo) records the
 * winner as h * W + w within its plane (or -1, see CAFFE_POOL_RELU_INPUT);
 * the backward pass sends each top_diff element to that position and sums
 * what arrives (overwriting bottom_diff).  pad must be smaller than the
 * kernel.
 *
 * Local response normalisation across channels:
 *   s_c = k + (alpha / local_size) * sum_{c' in win(c)} bottom_{c'}^2
 *   top_c = bottom_c * s_c^(-beta)
 *   win(c) = c - (local_size-1)/2 ... c - (local_size-1)/2 + local_size - 1,
 *            clipped to [0, C) (the divisor stays local_size)
 * and the backward pass is its exact derivative:
 *   bottom_diff_c = top_diff_c s_c^(-beta)
 *       - (2 alpha beta / local_size) bottom_c sum_{c': c in win(c')} top_diff_c' top_c' / s_c'
 *
 * Conventions (memory, streams, errors, status codes) are those of
 * caffe_conv.h: caller-owned 16-byte-aligned device pointers, asynchronous
 * execution on `stream`, negative caffe_status on failure with nothing
 * enqueued, no atomics.  All blobs are float, N x C x H x W.
 */
#ifndef CAFFE_LAYERS_H
#define CAFFE_LAYERS_H

#include <stddef.h>
#include <stdint.h>

#include "caffe_conv.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct caffe_pool_desc {
    int32_t N, C, H, W;
    int32_t kernel_h, kernel_w, stride_h, stride_w, pad_h, pad_w;
} caffe_pool_desc;

typedef struct caffe_lrn_desc {
    int32_t N, C, H, W;
    int32_t local_size; /* >= 1 */
    float alpha, beta, k;
} caffe_lrn_desc;

/* Host-only. */
int caffe_pool_out_shape(const caffe_pool_desc* desc, int32_t* Ho, int32_t* Wo);

/* Flags of caffe_maxpool_forward. */
enum caffe_pool_flags {
    /* bottom is the output of a ReLU: a window whose maximum is not > 0
     * records mask -1 (no winner), so the backward pass also applies that
     * ReLU's backward (it routes nothing where the ReLU's output was 0).
     * top is unchanged. */
    CAFFE_POOL_RELU_INPUT = 1,
    /* caffe_pool_lrn_forward_into only: the LRN's float output is not
     * written (top may be NULL); its staged bf16 copy is.  For callers whose
     * only other reader of that output is the fused backward
     * (caffe_conv_backward_pool_lrn, caffe_lrn_pool_backward), which forms
     * it again from `pooled`. */
    CAFFE_POOL_LRN_STAGE_ONLY = 2,
    /* caffe_pool_lrn_forward and caffe_pool_lrn_forward_into only: mask
     * (an int32_t pointer by type) receives one byte per pooled value, the
     * winner's offset du * kernel_w + dv within its window (255: no winner)
     * instead of its plane index: a quarter of the bytes to write and read.
     * Only caffe_conv_backward_pool_lrn with CAFFE_BACKWARD_POOL_MASK_OFFSETS
     * reads such a mask.  CAFFE_ERR_UNSUPPORTED for windows of more than 255
     * taps. */
    CAFFE_POOL_MASK_OFFSETS = 4
};

/* mask may be NULL when no backward pass will follow; flags is a set of
 * caffe_pool_flags. */
int caffe_maxpool_forward(const caffe_pool_desc* desc, const float* bottom, float* top,
                          int32_t* mask, int32_t flags, void* stream);

int caffe_maxpool_backward(const caffe_pool_desc* desc, const float* top_diff,
                           const int32_t* mask, float* bottom_diff, void* stream);

int caffe_lrn_forward(const caffe_lrn_desc* desc, const float* bottom, float* top, void* stream);

/* top is the forward output for the same bottom. */
int caffe_lrn_backward(const caffe_lrn_desc* desc, const float* bottom, const float* top,
                       const float* top_diff, float* bottom_diff, void* stream);

/* Max pooling followed by LRN of the pooled blob (CaffeNet's glue after
 * conv1 and conv2).  `pool` describes the pooling of bottom; `lrn` must
 * describe its output (N, C, Ho, Wo).  pooled, mask and top are written as
 * caffe_maxpool_forward (with `flags`) followed by caffe_lrn_forward on
 * `pooled` write them (the same two kernels, back to back: the pooled blob is
 * an output the backward needs).  mask may be NULL.  The support conditions
 * are those of caffe_lrn_pool_backward, so that a forward this call accepts
 * has a fused backward; with N = 0 nothing is launched and the status says
 * whether a geometry is supported. */
int caffe_pool_lrn_forward(const caffe_pool_desc* pool, const caffe_lrn_desc* lrn,
                           const float* bottom, float* pooled, int32_t* mask, float* top,
                           int32_t flags, void* stream);

/* caffe_pool_lrn_forward whose LRN output (top, still written) also goes,
 * rounded to bf16 (nearest even), to the staged bottom of the convolution
 * `next` that takes it as input, border included, in next's forward
 * workspace (next_workspace, at least caffe_conv_workspace_size(next,
 * CAFFE_PASS_FORWARD) bytes): next's forward then takes
 * CAFFE_FORWARD_BOTTOM_STAGED (caffe_conv_forward_ex) and skips the pass
 * that would read top back and stage it.  next's N, C, H, W must be the
 * LRN's (CAFFE_ERR_INVALID_ARG); next must be in a bf16 mode with groups of
 * a multiple of 16 channels that need no padding, the LRN of size 3 or 5
 * (caffe_pool_lrn_stage_supported, else CAFFE_ERR_UNSUPPORTED). */
int caffe_pool_lrn_forward_into(const caffe_pool_desc* pool, const caffe_lrn_desc* lrn,
                                const float* bottom, float* pooled, int32_t* mask, float* top,
                                int32_t flags, const caffe_conv_desc* next, void* next_workspace,
                                size_t next_ws_bytes, void* stream);

/* 1 when caffe_pool_lrn_forward_into can stage for `next`, else 0.
 * Host-only. */
int caffe_pool_lrn_stage_supported(const caffe_pool_desc* pool, const caffe_lrn_desc* lrn,
                                   const caffe_conv_desc* next);

/* The backward of that pair in one pass: bottom_diff as caffe_lrn_backward
 * (pooled, top, top_diff) followed by caffe_maxpool_backward (with `mask`)
 * would write it, without storing the pooled gradient (each block stages the
 * pooled gradient of its input rows' covering windows in LDS).  top must be
 * the LRN's forward output for `pooled` (caffe_pool_lrn_forward's): the
 * pass forms it again from `pooled` as the forward kernel does, with the
 * same bits, instead of reading it.
 * CAFFE_ERR_UNSUPPORTED unless lrn->local_size is 3 or 5, W <= 256 and
 * min(Ho, (kernel_h - 1) / stride_h + 2) * Wo <= 256 (a block stages at most
 * 256 pooled positions, one per thread). */
int caffe_lrn_pool_backward(const caffe_pool_desc* pool, const caffe_lrn_desc* lrn,
                            const float* pooled, const float* top, const float* top_diff,
                            const int32_t* mask, float* bottom_diff, void* stream);

/* caffe_lrn_pool_backward with flags: CAFFE_BACKWARD_POOL_MASK_OFFSETS
 * (caffe_conv.h) reads `mask` as the bytes caffe_pool_lrn_forward writes
 * with CAFFE_POOL_MASK_OFFSETS (CAFFE_ERR_UNSUPPORTED for windows of more
 * than 255 taps); other flags are CAFFE_ERR_INVALID_ARG. */
int caffe_lrn_pool_backward_ex(const caffe_pool_desc* pool, const caffe_lrn_desc* lrn,
                               const float* pooled, const float* top, const float* top_diff,
                               const int32_t* mask, float* bottom_diff, int32_t flags,
                               void* stream);

/* The backward pass of a convolution layer whose output feeds max pooling
 * followed by LRN (CaffeNet's conv1 and conv2 with their glue): the layer's
 * top gradient is the glue's backward, caffe_lrn_pool_backward(pool, lrn,
 * pooled, lrn_top, lrn_top_diff, pool_mask), and the rest is
 * caffe_conv_backward(desc, that gradient, top, bottom, weight, bottom_diff,
 * weight_diff, bias_diff, accumulate, flags, ...) -- the same results,
 * without the top gradient ever stored in float.  `pool` must describe the
 * pooling of this layer's top (N, K, Ho, Wo) and `lrn` the pooled blob, with
 * the support conditions of caffe_lrn_pool_backward.  pool_mask holds the
 * winners of the forward pooling; with CAFFE_POOL_RELU_INPUT there the
 * gradient is already masked by the layer's ReLU (pass
 * CAFFE_BACKWARD_TOP_DIFF_MASKED), otherwise `top` is read for the mask when
 * desc->relu.  Workspace: caffe_conv_workspace_size with
 * CAFFE_PASS_BACKWARD_POOL_LRN.
 * In the bf16 modes with K / group a multiple of 16, the glue's backward
 * writes the bfloat16 staging of the top gradient (and the bias-gradient
 * partials of its float values) directly: one pass instead of writing the
 * float gradient and reading it back.  Otherwise the float gradient goes to
 * the workspace first. */
int caffe_conv_backward_pool_lrn(const caffe_conv_desc* desc, const caffe_pool_desc* pool,
                                 const caffe_lrn_desc* lrn, const float* pooled,
                                 const float* lrn_top, const float* lrn_top_diff,
                                 const int32_t* pool_mask, const float* top, const void* bottom,
                                 const void* weight, float* bottom_diff, float* weight_diff,
                                 float* bias_diff, int32_t accumulate, int32_t flags,
                                 void* workspace, size_t ws_bytes, void* stream);

/* caffe_conv_backward_pool_lrn with the weight-side outputs ordered on
 * weight_stream, as caffe_conv_backward_ex (caffe_conv.h) describes: the
 * glue's backward and the data gradient on `stream`, the weight and bias
 * gradients on weight_stream after the staging, the streams not joined. */
int caffe_conv_backward_pool_lrn_ex(const caffe_conv_desc* desc, const caffe_pool_desc* pool,
                                    const caffe_lrn_desc* lrn, const float* pooled,
                                    const float* lrn_top, const float* lrn_top_diff,
                                    const int32_t* pool_mask, const float* top,
                                    const void* bottom, const void* weight, float* bottom_diff,
                                    float* weight_diff, float* bias_diff, int32_t accumulate,
                                    int32_t flags, void* workspace, size_t ws_bytes, void* stream,
                                    void* weight_stream);

/* The backward pass of a rectified-linear layer (Sec. 3.2 lists ReLU among
 * Caffe's layers): bottom_diff[i] = top[i] > 0 ? top_diff[i] : 0 for
 * i < count, where top is the layer's forward output (a NaN top gives 0).
 * bottom_diff may be top_diff (in place).  A network uses it where a ReLU's
 * backward is not folded into a neighbouring layer's kernels, e.g. to mask a
 * convolution's top gradient once before its data and weight gradients run
 * as separate calls. */
int caffe_relu_backward(const float* top, const float* top_diff, float* bottom_diff,
                        int64_t count, void* stream);

/* out[i] = bfloat16(in[i]) rounded to nearest even, i < count.  The input for
 * CAFFE_BF16 convolutions. */
int caffe_cast_f32_to_bf16(const float* in, uint16_t* out, int64_t count, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* CAFFE_LAYERS_H */
