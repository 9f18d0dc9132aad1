// layers.hip -- the glue layers that sit between CaffeNet's convolutions
// (max pooling and across-channel local response normalisation, both in the
// paper's Sec. 3.2 list of layer types) and the fp32 -> bf16 cast that feeds
// the bf16 convolution path.  All are HBM-bound elementwise/window kernels.
#include "device_common.h"
#include "kernels.h"

namespace caffe_hip {

// ----------------------------------------------------------------- max pool
// Window rows i*sh - ph .. + kh - 1 clipped to the image; the first maximum in
// row-major window order wins; mask holds its index h*W + w within the plane.
__global__ void __launch_bounds__(256)
maxpool_forward_kernel(const float* __restrict__ x, float* __restrict__ y,
                       int32_t* __restrict__ mask, int NC, int H, int W, int OH, int OW, int kh,
                       int kw, int sh, int sw, int ph, int pw)
{
    const long total = (long)NC * OH * OW;
    for (long e = blockIdx.x * (long)blockDim.x + threadIdx.x; e < total;
         e += (long)gridDim.x * blockDim.x) {
        const int j = (int)(e % OW);
        const int i = (int)((e / OW) % OH);
        const long nc = e / ((long)OH * OW);
        const float* plane = x + nc * H * W;
        int h0 = i * sh - ph, w0 = j * sw - pw;
        const int h1 = min(h0 + kh, H), w1 = min(w0 + kw, W);
        h0 = max(h0, 0);
        w0 = max(w0, 0);
        int best = h0 * W + w0;
        float bv = plane[best];
        for (int h = h0; h < h1; ++h)
            for (int w = w0; w < w1; ++w) {
                const float v = plane[h * W + w];
                if (v > bv) {
                    bv = v;
                    best = h * W + w;
                }
            }
        y[e] = bv;
        if (mask)
            mask[e] = best;
    }
}

// Gather form (one thread per input element, outputs visited in row-major
// order): deterministic, no atomics.
__global__ void __launch_bounds__(256)
maxpool_backward_kernel(const float* __restrict__ dy, const int32_t* __restrict__ mask,
                        float* __restrict__ dx, int NC, int H, int W, int OH, int OW, int kh,
                        int kw, int sh, int sw, int ph, int pw)
{
    const long total = (long)NC * H * W;
    for (long e = blockIdx.x * (long)blockDim.x + threadIdx.x; e < total;
         e += (long)gridDim.x * blockDim.x) {
        const int w = (int)(e % W);
        const int h = (int)((e / W) % H);
        const long nc = e / ((long)H * W);
        // outputs whose window covers (h, w): i*sh - ph <= h <= i*sh - ph + kh - 1
        const int i0 = max(0, (h + ph - kh + sh) / sh);
        const int i1 = min(OH - 1, (h + ph) / sh);
        const int j0 = max(0, (w + pw - kw + sw) / sw);
        const int j1 = min(OW - 1, (w + pw) / sw);
        const int self = h * W + w;
        const long obase = nc * OH * OW;
        float s = 0.f;
        for (int i = i0; i <= i1; ++i)
            for (int j = j0; j <= j1; ++j)
                if (mask[obase + i * OW + j] == self)
                    s += dy[obase + i * OW + j];
        dx[e] = s;
    }
}

static unsigned grid_for(long total)
{
    long b = (total + 255) / 256;
    return (unsigned)(b > 16384 ? 16384 : (b < 1 ? 1 : b));
}

hipError_t launch_maxpool_forward(const float* x, float* y, int32_t* mask, int NC, int H, int W,
                                  int OH, int OW, int kh, int kw, int sh, int sw, int ph, int pw,
                                  hipStream_t s)
{
    const long total = (long)NC * OH * OW;
    if (total == 0)
        return hipSuccess;
    hipLaunchKernelGGL(maxpool_forward_kernel, dim3(grid_for(total)), dim3(256), 0, s, x, y, mask,
                       NC, H, W, OH, OW, kh, kw, sh, sw, ph, pw);
    return hipGetLastError();
}

hipError_t launch_maxpool_backward(const float* dy, const int32_t* mask, float* dx, int NC, int H,
                                   int W, int OH, int OW, int kh, int kw, int sh, int sw, int ph,
                                   int pw, hipStream_t s)
{
    const long total = (long)NC * H * W;
    if (total == 0)
        return hipSuccess;
    hipLaunchKernelGGL(maxpool_backward_kernel, dim3(grid_for(total)), dim3(256), 0, s, dy, mask,
                       dx, NC, H, W, OH, OW, kh, kw, sh, sw, ph, pw);
    return hipGetLastError();
}

// ---------------------------------------------------------------------- LRN
// s_c = k + alpha/size * sum_{c' in win(c)} a_{c'}^2,  b_c = a_c s_c^-beta,
// win(c) = [c - (size-1)/2, c - (size-1)/2 + size - 1] clipped to [0, C).
__device__ __forceinline__ float lrn_scale(const float* col, int C, int HW, int c, int size,
                                           float alpha_over_n, float k)
{
    const int lo = max(0, c - (size - 1) / 2);
    const int hi = min(C, c - (size - 1) / 2 + size);
    float sq = 0.f;
    for (int q = lo; q < hi; ++q) {
        const float a = col[(long)q * HW];
        sq += a * a;
    }
    return k + alpha_over_n * sq;
}

__global__ void __launch_bounds__(256)
lrn_forward_kernel(const float* __restrict__ x, float* __restrict__ y, int N, int C, int HW,
                   int size, float alpha, float beta, float k)
{
    const long total = (long)N * C * HW;
    const float an = alpha / size;
    for (long e = blockIdx.x * (long)blockDim.x + threadIdx.x; e < total;
         e += (long)gridDim.x * blockDim.x) {
        const int pix = (int)(e % HW);
        const int c = (int)((e / HW) % C);
        const long n = e / ((long)C * HW);
        const float* col = x + n * C * HW + pix;
        const float s = lrn_scale(col, C, HW, c, size, an, k);
        y[e] = col[(long)c * HW] * powf(s, -beta);
    }
}

// dx_c = g_c s_c^-beta - (2 alpha beta / size) a_c sum_{c': c in win(c')} g_c' b_c' / s_c'
__global__ void __launch_bounds__(256)
lrn_backward_kernel(const float* __restrict__ x, const float* __restrict__ y,
                    const float* __restrict__ dy, float* __restrict__ dx, int N, int C, int HW,
                    int size, float alpha, float beta, float k)
{
    const long total = (long)N * C * HW;
    const float an = alpha / size;
    const int pre = (size - 1) / 2;
    for (long e = blockIdx.x * (long)blockDim.x + threadIdx.x; e < total;
         e += (long)gridDim.x * blockDim.x) {
        const int pix = (int)(e % HW);
        const int c = (int)((e / HW) % C);
        const long n = e / ((long)C * HW);
        const long cb = n * C * HW + pix;
        const float* col = x + cb;
        const float s_c = lrn_scale(col, C, HW, c, size, an, k);
        const int q0 = max(0, c + pre - size + 1);
        const int q1 = min(C - 1, c + pre);
        float cross = 0.f;
        for (int q = q0; q <= q1; ++q) {
            const float s_q = lrn_scale(col, C, HW, q, size, an, k);
            cross += dy[cb + (long)q * HW] * y[cb + (long)q * HW] / s_q;
        }
        dx[e] = dy[e] * powf(s_c, -beta) - 2.f * an * beta * col[(long)c * HW] * cross;
    }
}

hipError_t launch_lrn_forward(const float* x, float* y, int N, int C, int HW, int size,
                              float alpha, float beta, float k, hipStream_t s)
{
    const long total = (long)N * C * HW;
    if (total == 0)
        return hipSuccess;
    hipLaunchKernelGGL(lrn_forward_kernel, dim3(grid_for(total)), dim3(256), 0, s, x, y, N, C, HW,
                       size, alpha, beta, k);
    return hipGetLastError();
}

hipError_t launch_lrn_backward(const float* x, const float* y, const float* dy, float* dx, int N,
                               int C, int HW, int size, float alpha, float beta, float k,
                               hipStream_t s)
{
    const long total = (long)N * C * HW;
    if (total == 0)
        return hipSuccess;
    hipLaunchKernelGGL(lrn_backward_kernel, dim3(grid_for(total)), dim3(256), 0, s, x, y, dy, dx,
                       N, C, HW, size, alpha, beta, k);
    return hipGetLastError();
}

// --------------------------------------------------------------------- cast
__global__ void __launch_bounds__(256)
cast_f32_bf16_kernel(const float* __restrict__ x, uint16_t* __restrict__ y, int64_t count)
{
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < count;
         e += (int64_t)gridDim.x * blockDim.x)
        y[e] = f32_to_bf16_rne(x[e]);
}

hipError_t launch_cast_f32_bf16(const float* x, uint16_t* y, int64_t count, hipStream_t s)
{
    if (count == 0)
        return hipSuccess;
    hipLaunchKernelGGL(cast_f32_bf16_kernel, dim3(grid_for(count)), dim3(256), 0, s, x, y, count);
    return hipGetLastError();
}

}  // namespace caffe_hip
