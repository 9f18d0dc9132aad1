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
    const int total = NC * OH * OW;  // every tensor holds < 2^31 bytes
    const int e = blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= total)
        return;
    const int j = e % OW;
    const int t = e / OW;
    const int i = t % OH;
    const int nc = t / OH;
    const float* plane = x + nc * (H * W);
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

// Gather form (one thread per input element, outputs visited in row-major
// order): deterministic, no atomics.
__global__ void __launch_bounds__(256)
maxpool_backward_kernel(const float* __restrict__ dy, const int32_t* __restrict__ mask,
                        float* __restrict__ dx, int NC, int H, int W, int OH, int OW, int kh,
                        int kw, int sh, int sw, int ph, int pw)
{
    const int total = NC * H * W;
    const int e = blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= total)
        return;
    const int w = e % W;
    const int t = e / W;
    const int h = t % H;
    const int nc = t / H;
    // outputs whose window covers (h, w): i*sh - ph <= h <= i*sh - ph + kh - 1
    const int i0 = max(0, (h + ph - kh + sh) / sh);
    const int i1 = min(OH - 1, (h + ph) / sh);
    const int j0 = max(0, (w + pw - kw + sw) / sw);
    const int j1 = min(OW - 1, (w + pw) / sw);
    const int self = h * W + w;
    const int obase = nc * (OH * OW);
    float s = 0.f;
    for (int i = i0; i <= i1; ++i)
        for (int j = j0; j <= j1; ++j)
            if (mask[obase + i * OW + j] == self)
                s += dy[obase + i * OW + j];
    dx[e] = s;
}

static unsigned grid_for(long total)
{
    long b = (total + 255) / 256;
    return (unsigned)(b > 16384 ? 16384 : (b < 1 ? 1 : b));
}

static unsigned grid_exact(long total) { return (unsigned)((total + 255) / 256); }

hipError_t launch_maxpool_forward(const float* x, float* y, int32_t* mask, int NC, int H, int W,
                                  int OH, int OW, int kh, int kw, int sh, int sw, int ph, int pw,
                                  hipStream_t s)
{
    const long total = (long)NC * OH * OW;
    if (total == 0)
        return hipSuccess;
    hipLaunchKernelGGL(maxpool_forward_kernel, dim3(grid_exact(total)), dim3(256), 0, s, x, y, mask,
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
    hipLaunchKernelGGL(maxpool_backward_kernel, dim3(grid_exact(total)), dim3(256), 0, s, dy, mask,
                       dx, NC, H, W, OH, OW, kh, kw, sh, sw, ph, pw);
    return hipGetLastError();
}

// ---------------------------------------------------------------------- LRN
// s_c = k + alpha/size * sum_{c' in win(c)} a_{c'}^2,  b_c = a_c s_c^-beta,
// win(c) = [c - pre, c - pre + size - 1] clipped to [0, C), pre = (size-1)/2.
//
// One thread per (n, pixel) column walks the channels; lanes run along the
// pixels, so every load is coalesced and every input is read once.  The
// window's squares live in a register ring of SIZE entries and each sum is
// re-added from the ring (no running add/subtract, so no drift).
template <int SIZE>
__global__ void __launch_bounds__(256)
lrn_forward_kernel(const float* __restrict__ x, float* __restrict__ y, int N, int C, int HW,
                   float alpha_over_n, float beta, float k)
{
    constexpr int PRE = (SIZE - 1) / 2;
    constexpr int POST = SIZE - 1 - PRE;
    const int e = blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= N * HW)
        return;
    const int n = e / HW;
    const int pix = e - n * HW;
    const float* col = x + n * C * HW + pix;
    float* out = y + n * C * HW + pix;
    float a[SIZE];  // a[q] = value of channel c - PRE + q (0 outside)
#pragma unroll
    for (int q = 0; q < SIZE; ++q) {
        const int ch = q - PRE;
        a[q] = (ch >= 0 && ch < C) ? col[ch * HW] : 0.f;
    }
    for (int c = 0; c < C; ++c) {
        float sq = 0.f;
#pragma unroll
        for (int q = 0; q < SIZE; ++q)
            sq += a[q] * a[q];
        const float s = k + alpha_over_n * sq;
        out[c * HW] = a[PRE] * powf(s, -beta);
#pragma unroll
        for (int q = 0; q + 1 < SIZE; ++q)
            a[q] = a[q + 1];
        const int nxt = c + 1 + POST;
        a[SIZE - 1] = nxt < C ? col[nxt * HW] : 0.f;
    }
}

// dx_c = g_c s_c^-beta - (2 alpha beta / size) a_c sum_{c': c in win(c')} g_c' b_c' / s_c'
// c in win(c') <=> c' in [c - POST, c + PRE].  Step j computes s_j and the
// ratio r_j = g_j b_j / s_j, then emits dx for c = j - PRE.
template <int SIZE>
__global__ void __launch_bounds__(256)
lrn_backward_kernel(const float* __restrict__ x, const float* __restrict__ y,
                    const float* __restrict__ dy, float* __restrict__ dx, int N, int C, int HW,
                    float alpha_over_n, float beta, float k)
{
    constexpr int PRE = (SIZE - 1) / 2;
    constexpr int POST = SIZE - 1 - PRE;
    const int e = blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= N * HW)
        return;
    const int n = e / HW;
    const int pix = e - n * HW;
    const int base = n * C * HW + pix;
    float a[SIZE];          // inputs of channels j - PRE .. j + POST
    float r[SIZE];          // ratios of channels j - SIZE + 1 .. j
    float sc[PRE + 1];      // s of channels j - PRE .. j
    float ac[PRE + 1];      // inputs of channels j - PRE .. j
    float gc[PRE + 1];      // gradients of channels j - PRE .. j
#pragma unroll
    for (int q = 0; q < SIZE; ++q) {
        const int ch = q - PRE;
        a[q] = (ch >= 0 && ch < C) ? x[base + ch * HW] : 0.f;
        r[q] = 0.f;
    }
#pragma unroll
    for (int q = 0; q <= PRE; ++q)
        sc[q] = ac[q] = gc[q] = 0.f;
    const float coef = 2.f * alpha_over_n * beta;
    for (int j = 0; j < C + PRE; ++j) {
        float s = 1.f, g = 0.f, rj = 0.f;
        if (j < C) {
            float sq = 0.f;
#pragma unroll
            for (int q = 0; q < SIZE; ++q)
                sq += a[q] * a[q];
            s = k + alpha_over_n * sq;
            g = dy[base + j * HW];
            rj = g * y[base + j * HW] / s;
        }
#pragma unroll
        for (int q = 0; q + 1 < SIZE; ++q)
            r[q] = r[q + 1];
        r[SIZE - 1] = rj;
#pragma unroll
        for (int q = 0; q < PRE; ++q) {
            sc[q] = sc[q + 1];
            ac[q] = ac[q + 1];
            gc[q] = gc[q + 1];
        }
        sc[PRE] = s;
        ac[PRE] = a[PRE];
        gc[PRE] = g;
        const int c = j - PRE;
        if (c >= 0) {
            float cross = 0.f;  // r of channels c - POST .. c + PRE = j - SIZE + 1 .. j
#pragma unroll
            for (int q = 0; q < SIZE; ++q)
                cross += r[q];
            dx[base + c * HW] = gc[0] * powf(sc[0], -beta) - coef * ac[0] * cross;
        }
#pragma unroll
        for (int q = 0; q + 1 < SIZE; ++q)
            a[q] = a[q + 1];
        const int nxt = j + 1 + POST;
        a[SIZE - 1] = nxt < C ? x[base + nxt * HW] : 0.f;
    }
}

// Any window size: direct evaluation, one thread per element.
__device__ __forceinline__ float lrn_scale(const float* col, int C, int HW, int c, int size,
                                           float alpha_over_n, float k)
{
    const int lo = max(0, c - (size - 1) / 2);
    const int hi = min(C, c - (size - 1) / 2 + size);
    float sq = 0.f;
    for (int q = lo; q < hi; ++q) {
        const float a = col[q * HW];
        sq += a * a;
    }
    return k + alpha_over_n * sq;
}

__global__ void __launch_bounds__(256)
lrn_forward_any_kernel(const float* __restrict__ x, float* __restrict__ y, int N, int C, int HW,
                       int size, float alpha_over_n, float beta, float k)
{
    const int e = blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= N * C * HW)
        return;
    const int pix = e % HW;
    const int c = (e / HW) % C;
    const int n = e / (C * HW);
    const float* col = x + n * C * HW + pix;
    const float s = lrn_scale(col, C, HW, c, size, alpha_over_n, k);
    y[e] = col[c * HW] * powf(s, -beta);
}

__global__ void __launch_bounds__(256)
lrn_backward_any_kernel(const float* __restrict__ x, const float* __restrict__ y,
                        const float* __restrict__ dy, float* __restrict__ dx, int N, int C,
                        int HW, int size, float alpha_over_n, float beta, float k)
{
    const int e = blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= N * C * HW)
        return;
    const int pre = (size - 1) / 2;
    const int pix = e % HW;
    const int c = (e / HW) % C;
    const int n = e / (C * HW);
    const int cb = n * C * HW + pix;
    const float* col = x + cb;
    const float s_c = lrn_scale(col, C, HW, c, size, alpha_over_n, k);
    const int q0 = max(0, c + pre - size + 1);
    const int q1 = min(C - 1, c + pre);
    float cross = 0.f;
    for (int q = q0; q <= q1; ++q) {
        const float s_q = lrn_scale(col, C, HW, q, size, alpha_over_n, k);
        cross += dy[cb + q * HW] * y[cb + q * HW] / s_q;
    }
    dx[e] = dy[e] * powf(s_c, -beta) - 2.f * alpha_over_n * beta * col[c * HW] * cross;
}

hipError_t launch_lrn_forward(const float* x, float* y, int N, int C, int HW, int size,
                              float alpha, float beta, float k, hipStream_t s)
{
    const long cols = (long)N * HW;
    if (cols == 0)
        return hipSuccess;
    const float an = alpha / size;
    if (size == 5)
        hipLaunchKernelGGL(lrn_forward_kernel<5>, dim3(grid_exact(cols)), dim3(256), 0, s, x, y,
                           N, C, HW, an, beta, k);
    else if (size == 3)
        hipLaunchKernelGGL(lrn_forward_kernel<3>, dim3(grid_exact(cols)), dim3(256), 0, s, x, y,
                           N, C, HW, an, beta, k);
    else
        hipLaunchKernelGGL(lrn_forward_any_kernel, dim3(grid_exact(cols * C)), dim3(256), 0, s, x,
                           y, N, C, HW, size, an, beta, k);
    return hipGetLastError();
}

hipError_t launch_lrn_backward(const float* x, const float* y, const float* dy, float* dx, int N,
                               int C, int HW, int size, float alpha, float beta, float k,
                               hipStream_t s)
{
    const long cols = (long)N * HW;
    if (cols == 0)
        return hipSuccess;
    const float an = alpha / size;
    if (size == 5)
        hipLaunchKernelGGL(lrn_backward_kernel<5>, dim3(grid_exact(cols)), dim3(256), 0, s, x, y,
                           dy, dx, N, C, HW, an, beta, k);
    else if (size == 3)
        hipLaunchKernelGGL(lrn_backward_kernel<3>, dim3(grid_exact(cols)), dim3(256), 0, s, x, y,
                           dy, dx, N, C, HW, an, beta, k);
    else
        hipLaunchKernelGGL(lrn_backward_any_kernel, dim3(grid_exact(cols * C)), dim3(256), 0, s,
                           x, y, dy, dx, N, C, HW, size, an, beta, k);
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
