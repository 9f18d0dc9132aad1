// conv_aux.hip -- the HBM-bound helpers of the convolution layer's backward
// pass: the fused ReLU backward + bias-gradient partial sums, the weight
// re-layout for the phase-stacked data gradient, and the fixed-order
// reduction of the split-K weight-gradient partials.
#include "device_common.h"
#include "kernels.h"

namespace caffe_hip {

// One wave per (n, k) plane: D = relu ? G [Y > 0] : G, and the plane's sum
// (the per-image bias-gradient term sum_{i,j} D[n,k,i,j]) in a fixed order:
// lane-strided partial sums, then a butterfly across the wave.
__global__ void __launch_bounds__(256)
relu_mask_bias_kernel(const float* __restrict__ G, const float* __restrict__ Y,
                      float* __restrict__ D, float* __restrict__ plane_sums, int planes,
                      int plane_size, int relu)
{
    const int lane = threadIdx.x & 63;
    const int wave = (blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    const int nwaves = (gridDim.x * blockDim.x) >> 6;
    for (int pl = wave; pl < planes; pl += nwaves) {
        const size_t base = (size_t)pl * plane_size;
        float s = 0.f;
        for (int e = lane; e < plane_size; e += 64) {
            float d = G[base + e];
            if (relu && !(Y[base + e] > 0.f))
                d = 0.f;
            if (D)
                D[base + e] = d;
            s += d;
        }
        s = wave_sum(s);
        if (plane_sums && lane == 0)
            plane_sums[pl] = s;
    }
}

hipError_t launch_relu_mask_bias(const float* G, const float* Y, float* D, float* plane_sums,
                                 int planes, int plane_size, int relu, hipStream_t s)
{
    if (planes == 0)
        return hipSuccess;
    const int waves_per_block = 4;
    int blocks = (planes + waves_per_block - 1) / waves_per_block;
    if (blocks > 8192)
        blocks = 8192;
    hipLaunchKernelGGL(relu_mask_bias_kernel, dim3(blocks), dim3(64 * waves_per_block), 0, s, G,
                       Y, D, plane_sums, planes, plane_size, relu);
    return hipGetLastError();
}

// Wt[g][m = (c, fh, fw)][r = (k, th, tw)]
//   = W[g*Kg + k][c][fh + sh*(Th-1-th)][fw + sw*(Tw-1-tw)], 0 past the kernel edge.
__global__ void __launch_bounds__(256)
dgrad_weight_transform_kernel(const float* __restrict__ W, float* __restrict__ Wt, int G, int Kg,
                              int Cg, int kh, int kw, int sh, int sw, int Th, int Tw)
{
    const int Mt = Cg * sh * sw;
    const int Rt = Kg * Th * Tw;
    const long total = (long)G * Mt * Rt;
    for (long e = blockIdx.x * (long)blockDim.x + threadIdx.x; e < total;
         e += (long)gridDim.x * blockDim.x) {
        const int r = (int)(e % Rt);
        const long gm = e / Rt;
        const int m = (int)(gm % Mt);
        const int g = (int)(gm / Mt);
        const int k = r / (Th * Tw);
        const int t = r - k * Th * Tw;
        const int th = t / Tw, tw = t - th * Tw;
        const int c = m / (sh * sw);
        const int f = m - c * sh * sw;
        const int fh = f / sw, fw = f - fh * sw;
        const int u = fh + sh * (Th - 1 - th);
        const int v = fw + sw * (Tw - 1 - tw);
        float val = 0.f;
        if (u < kh && v < kw)
            val = W[(((long)(g * Kg + k) * Cg + c) * kh + u) * kw + v];
        Wt[e] = val;
    }
}

hipError_t launch_dgrad_weight_transform(const float* W, float* Wt, int G, int Kg, int Cg, int kh,
                                         int kw, int sh, int sw, int Th, int Tw, hipStream_t s)
{
    const long total = (long)G * Cg * sh * sw * Kg * Th * Tw;
    if (total == 0)
        return hipSuccess;
    long blocks = (total + 255) / 256;
    if (blocks > 4096)
        blocks = 4096;
    hipLaunchKernelGGL(dgrad_weight_transform_kernel, dim3((unsigned)blocks), dim3(256), 0, s, W,
                       Wt, G, Kg, Cg, kh, kw, sh, sw, Th, Tw);
    return hipGetLastError();
}

// Fixed-order sums: out[i] = (acc ? out[i] : 0) + P[0][i] + P[1][i] + ...,
// db[k] = (acc ? db[k] : 0) + sums[0*K + k] + sums[1*K + k] + ...
__global__ void __launch_bounds__(256)
wgrad_reduce_kernel(const float* __restrict__ P, float* __restrict__ out, int count, int splits,
                    const float* __restrict__ plane_sums, float* __restrict__ db, int N, int K,
                    int accumulate)
{
    const int total = count + (db ? K : 0);
    for (int e = blockIdx.x * blockDim.x + threadIdx.x; e < total; e += gridDim.x * blockDim.x) {
        if (e < count) {
            float s = 0.f;
            for (int q = 0; q < splits; ++q)
                s += P[(size_t)q * count + e];
            out[e] = accumulate ? out[e] + s : s;
        } else {
            const int k = e - count;
            float s = 0.f;
            for (int n = 0; n < N; ++n)
                s += plane_sums[(size_t)n * K + k];
            db[k] = accumulate ? db[k] + s : s;
        }
    }
}

hipError_t launch_wgrad_reduce(const float* P, float* out, int count, int splits,
                               const float* plane_sums, float* db, int N, int K, int accumulate,
                               hipStream_t s)
{
    const int total = count + (db ? K : 0);
    if (total == 0)
        return hipSuccess;
    int blocks = (total + 255) / 256;
    if (blocks > 4096)
        blocks = 4096;
    hipLaunchKernelGGL(wgrad_reduce_kernel, dim3(blocks), dim3(256), 0, s, P, out, count, splits,
                       plane_sums, db, N, K, accumulate);
    return hipGetLastError();
}

__global__ void __launch_bounds__(256) fill_zero_kernel(float* __restrict__ out, int64_t count)
{
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < count;
         e += (int64_t)gridDim.x * blockDim.x)
        out[e] = 0.f;
}

hipError_t launch_fill_zero(float* out, int64_t count, hipStream_t s)
{
    if (count == 0)
        return hipSuccess;
    int64_t blocks = (count + 255) / 256;
    if (blocks > 4096)
        blocks = 4096;
    hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)blocks), dim3(256), 0, s, out, count);
    return hipGetLastError();
}

}  // namespace caffe_hip
