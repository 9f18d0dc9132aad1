// solver.hip -- the softmax loss layer (forward and backward in one pass)
// and the SGD parameter update.  Both are HBM-bound: one read of the scores
// and one write of each wanted output; one read of w, g, v and one write of
// w, v.
#include "device_common.h"
#include "kernels.h"

namespace caffe_hip {

__device__ __forceinline__ float wave_max(float v)
{
    for (int off = 32; off > 0; off >>= 1)
        v = fmaxf(v, __shfl_xor(v, off, 64));
    return v;
}

// One wave per sample: the row maximum, the sum of exponentials (lane-strided
// partial sums in index order, then a butterfly), the sample's loss, and the
// probabilities / gradient row.
__global__ void __launch_bounds__(256)
softmax_loss_rows_kernel(const float* __restrict__ z, const int32_t* __restrict__ labels, int N,
                         int K, float loss_weight, float* __restrict__ sample_loss,
                         float* __restrict__ prob, float* __restrict__ diff)
{
    const int lane = threadIdx.x & 63;
    const int n = (blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    if (n >= N)
        return;
    const float* row = z + (size_t)n * K;
    float m = -INFINITY;
    for (int k = lane; k < K; k += 64)
        m = fmaxf(m, row[k]);
    m = wave_max(m);
    float s = 0.f;
    for (int k = lane; k < K; k += 64)
        s += expf(row[k] - m);
    s = wave_sum(s);
    const int y = labels[n];
    const bool ok = y >= 0 && y < K;
    if (lane == 0)
        sample_loss[n] = ok ? logf(s) - (row[y] - m) : NAN;
    if (prob || diff) {
        const float inv_s = 1.f / s;
        const float scale = loss_weight / (float)N;
        for (int k = lane; k < K; k += 64) {
            const float p = expf(row[k] - m) * inv_s;
            if (prob)
                prob[(size_t)n * K + k] = p;
            if (diff)
                diff[(size_t)n * K + k] = (p - (k == y ? 1.f : 0.f)) * scale;
        }
    }
}

// loss = loss_weight * sum_n sample_loss[n] / N in a fixed order: thread t
// adds samples t, t + 256, ... in order, then the 256 partial sums are added
// pairwise in a fixed tree.
__global__ void __launch_bounds__(256)
softmax_loss_total_kernel(const float* __restrict__ sample_loss, int N, float loss_weight,
                          float* __restrict__ loss)
{
    __shared__ float part[256];
    float s = 0.f;
    for (int n = threadIdx.x; n < N; n += 256)
        s += sample_loss[n];
    part[threadIdx.x] = s;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w)
            part[threadIdx.x] += part[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0)
        *loss = N > 0 ? loss_weight * part[0] / (float)N : 0.f;
}

hipError_t launch_softmax_loss(const float* z, const int32_t* labels, int N, int K,
                               float loss_weight, float* loss, float* sample_loss, float* prob,
                               float* diff, hipStream_t s)
{
    if (N > 0)
        hipLaunchKernelGGL(softmax_loss_rows_kernel, dim3((N + 3) / 4), dim3(256), 0, s, z,
                           labels, N, K, loss_weight, sample_loss, prob, diff);
    hipLaunchKernelGGL(softmax_loss_total_kernel, dim3(1), dim3(256), 0, s, sample_loss, N,
                       loss_weight, loss);
    return hipGetLastError();
}

// v <- momentum v + lr (g + decay w); w <- w - v, four elements per lane per
// iteration (the pointers are 16-byte aligned), then the tail.  With lr_dev
// non-null the rate is read from device memory when the kernel runs.
__global__ void __launch_bounds__(256)
sgd_update_kernel(float* __restrict__ w, const float* __restrict__ g, float* __restrict__ v,
                  int64_t count, float lr_arg, const float* __restrict__ lr_dev, float momentum,
                  float decay)
{
    const float lr = lr_dev ? *lr_dev : lr_arg;
    const int64_t n4 = count >> 2;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n4; i += stride) {
        float4 wv = reinterpret_cast<float4*>(w)[i];
        const float4 gv = reinterpret_cast<const float4*>(g)[i];
        float4 hv = reinterpret_cast<float4*>(v)[i];
        hv.x = momentum * hv.x + lr * (gv.x + decay * wv.x);
        hv.y = momentum * hv.y + lr * (gv.y + decay * wv.y);
        hv.z = momentum * hv.z + lr * (gv.z + decay * wv.z);
        hv.w = momentum * hv.w + lr * (gv.w + decay * wv.w);
        wv.x -= hv.x;
        wv.y -= hv.y;
        wv.z -= hv.z;
        wv.w -= hv.w;
        reinterpret_cast<float4*>(v)[i] = hv;
        reinterpret_cast<float4*>(w)[i] = wv;
    }
    for (int64_t i = (n4 << 2) + blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < count;
         i += stride) {
        const float h = momentum * v[i] + lr * (g[i] + decay * w[i]);
        v[i] = h;
        w[i] -= h;
    }
}

hipError_t launch_sgd_update(float* w, const float* g, float* v, int64_t count, float lr,
                             const float* lr_dev, float momentum, float decay, hipStream_t s)
{
    if (count == 0)
        return hipSuccess;
    int64_t blocks = ((count >> 2) + 255) / 256;
    blocks = blocks < 1 ? 1 : (blocks > 4096 ? 4096 : blocks);
    hipLaunchKernelGGL(sgd_update_kernel, dim3((unsigned)blocks), dim3(256), 0, s, w, g, v, count,
                       lr, lr_dev, momentum, decay);
    return hipGetLastError();
}

}  // namespace caffe_hip
