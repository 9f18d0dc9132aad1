/*
 * caffe_solver.h -- C ABI of the softmax loss layer and of the stochastic
 * gradient descent update, in the same library as caffe_conv.h
 * (libcaffe_conv.so).
 *
 * The paper lists softmax loss among Caffe's layer types (Sec. 3.2): the
 * loss layer that ends a network and produces the objective and its
 * gradient.  It trains networks by stochastic gradient descent over
 * mini-batches, with learning-rate decay schedules and momentum (Sec. 3.4,
 * Fig. 1's LeNet).  It gives no formulas; the library computes:
 *
 * Softmax loss of N score vectors z_n of K classes (row n of an N x K float
 * array, e.g. an N x K x 1 x 1 blob) with int32 labels y_n in [0, K):
 *   m_n = max_k z_{n,k},  s_n = sum_k exp(z_{n,k} - m_n)
 *   p_{n,k} = exp(z_{n,k} - m_n) / s_n
 *   sample_loss_n = log s_n - (z_{n,y_n} - m_n)          (= -log p_{n,y_n})
 *   loss = loss_weight * (sum_n sample_loss_n) / N
 *   scores_diff_{n,k} = loss_weight * (p_{n,k} - [k == y_n]) / N
 * The batch sum runs in a fixed order (bitwise reproducible).  A label
 * outside [0, K) makes that sample's loss (and so `loss`) NaN and leaves the
 * -1 term out of its gradient row; labels are not checked on the host.
 *
 * SGD update of one parameter blob w (count floats) with its gradient g and
 * momentum history v, at learning rate lr:
 *   v <- momentum * v + lr * (g + weight_decay * w)
 *   w <- w - v
 * (momentum 0 and weight_decay 0 give plain gradient descent).  Every
 * parameter blob of a network takes its own call (per-blob rates, e.g. a
 * bias multiplier, are the caller's lr).
 *
 * Learning-rate schedules at iteration t >= 0 (0 for the first update),
 * evaluated on the host in double precision:
 *   CAFFE_LR_FIXED  base_lr
 *   CAFFE_LR_STEP   base_lr * gamma^floor(t / stepsize)
 *   CAFFE_LR_EXP    base_lr * gamma^t
 *   CAFFE_LR_INV    base_lr * (1 + gamma * t)^(-power)
 *
 * Conventions (memory, streams, errors, status codes) are those of
 * caffe_conv.h: caller-owned 16-byte-aligned device pointers, asynchronous
 * execution on `stream`, negative caffe_status on failure with nothing
 * enqueued, no atomics.
 */
#ifndef CAFFE_SOLVER_H
#define CAFFE_SOLVER_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum caffe_lr_policy {
    CAFFE_LR_FIXED = 0,
    CAFFE_LR_STEP = 1,
    CAFFE_LR_EXP = 2,
    CAFFE_LR_INV = 3
};

typedef struct caffe_lr_schedule {
    int32_t policy;   /* a caffe_lr_policy */
    float base_lr;    /* >= 0 */
    float gamma;      /* step, exp: the decay factor; inv: the rate in (1 + gamma t) */
    float power;      /* inv only */
    int32_t stepsize; /* step only, >= 1 */
} caffe_lr_schedule;

/* Host-only: *lr = the schedule's rate at iteration `iter` (>= 0).
 * CAFFE_ERR_INVALID_ARG for an unknown policy, a negative base rate or
 * iteration, a step schedule with stepsize < 1, or a rate that is not finite
 * (e.g. inv with 1 + gamma t <= 0). */
int caffe_sgd_learning_rate(const caffe_lr_schedule* schedule, int64_t iter, float* lr);

/* Softmax loss forward and backward in one pass.  scores: N x K floats;
 * labels: N int32; loss: 1 float (written); sample_loss: N floats (written,
 * the per-sample losses the total is summed from); prob and scores_diff:
 * N x K floats each, or NULL when not wanted.  N >= 0 (N = 0 writes
 * loss = 0), 1 <= K <= 2^24; N * K * 4 < 2^31. */
int caffe_softmax_loss(const float* scores, const int32_t* labels, int32_t N, int32_t K,
                       float loss_weight, float* loss, float* sample_loss, float* prob,
                       float* scores_diff, void* stream);

/* SGD with momentum and L2 weight decay, in place on w and v (count floats
 * each, count >= 0; g is read only).  w, g and v must not overlap. */
int caffe_sgd_update(float* w, const float* g, float* v, int64_t count, float lr, float momentum,
                     float weight_decay, void* stream);

/* The same update with the learning rate read from device memory (`lr`, one
 * float, 4-byte aligned) when the kernel runs, not when it is enqueued: a
 * captured HIP graph of a training iteration then follows a schedule when
 * the caller writes the iteration's rate to `lr` before each replay. */
int caffe_sgd_update_device_lr(float* w, const float* g, float* v, int64_t count, const float* lr,
                               float momentum, float weight_decay, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* CAFFE_SOLVER_H */
