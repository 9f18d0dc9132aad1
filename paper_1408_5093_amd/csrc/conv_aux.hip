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
        int e = lane;
        // four independent loads in flight per lane, summed in index order
        for (; e + 192 < plane_size; e += 256) {
            float d[4];
#pragma unroll
            for (int u = 0; u < 4; ++u)
                d[u] = G[base + e + 64 * u];
            if (relu) {
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    d[u] = Y[base + e + 64 * u] > 0.f ? d[u] : 0.f;
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                if (D)
                    D[base + e + 64 * u] = d[u];
                s += d[u];
            }
        }
        for (; e < plane_size; e += 64) {
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

// D = G [Y > 0], element by element (four per lane per iteration when all
// three pointers are 16-byte aligned).
__global__ void __launch_bounds__(256)
relu_mask_kernel(const float* __restrict__ G, const float* __restrict__ Y, float* __restrict__ D,
                 int64_t count, int vec)
{
    const int64_t n4 = vec ? count >> 2 : 0;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n4; i += stride) {
        const float4 g = reinterpret_cast<const float4*>(G)[i];
        const float4 y = reinterpret_cast<const float4*>(Y)[i];
        float4 d;
        d.x = y.x > 0.f ? g.x : 0.f;
        d.y = y.y > 0.f ? g.y : 0.f;
        d.z = y.z > 0.f ? g.z : 0.f;
        d.w = y.w > 0.f ? g.w : 0.f;
        reinterpret_cast<float4*>(D)[i] = d;
    }
    for (int64_t i = (n4 << 2) + blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < count;
         i += stride)
        D[i] = Y[i] > 0.f ? G[i] : 0.f;
}

hipError_t launch_relu_mask(const float* G, const float* Y, float* D, int64_t count, hipStream_t s)
{
    if (count == 0)
        return hipSuccess;
    int64_t blocks = ((count >> 2) + 255) / 256;
    blocks = std::max<int64_t>(1, std::min<int64_t>(blocks, 4096));
    const int vec = (((uintptr_t)G | (uintptr_t)Y | (uintptr_t)D) & 15) == 0;
    hipLaunchKernelGGL(relu_mask_kernel, dim3((unsigned)blocks), dim3(256), 0, s, G, Y, D, count,
                       vec);
    return hipGetLastError();
}

// Wt[g][r][m = (c, fh, fw)] = W[g*Kg + k][c][fh + sh*(Th-1-th)][fw + sw*(Tw-1-tw)],
// 0 past the kernel edge; r = (k, th, tw), or r = (k / tk, th, tw, k % tk)
// when tk > 0, or r = (th, tw, k) when tk < 0.  m is contiguous (the layout
// the GEMM copies into LDS).
__global__ void __launch_bounds__(256)
dgrad_weight_transform_kernel(const float* __restrict__ W, float* __restrict__ Wt, int G, int Kg,
                              int Cg, int kh, int kw, int sh, int sw, int Th, int Tw, int tk)
{
    const int Mt = Cg * sh * sw;
    const int Rt = Kg * Th * Tw;
    const long total = (long)G * Mt * Rt;
    for (long e = blockIdx.x * (long)blockDim.x + threadIdx.x; e < total;
         e += (long)gridDim.x * blockDim.x) {
        const int m = (int)(e % Mt);
        const long gr = e / Mt;
        const int r = (int)(gr % Rt);
        const int g = (int)(gr / Rt);
        int k, t;
        if (tk > 0) {  // r = (k / tk, th, tw, k % tk)
            const int ki = r % tk;
            t = (r / tk) % (Th * Tw);
            k = (r / (tk * Th * Tw)) * tk + ki;
        } else if (tk < 0) {  // r = (th, tw, k)
            t = r / Kg;
            k = r - t * Kg;
        } else {       // r = (k, th, tw)
            k = r / (Th * Tw);
            t = r - k * Th * Tw;
        }
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
                                         int kw, int sh, int sw, int Th, int Tw, int tk,
                                         hipStream_t s)
{
    const long total = (long)G * Cg * sh * sw * Kg * Th * Tw;
    if (total == 0)
        return hipSuccess;
    long blocks = (total + 255) / 256;
    if (blocks > 4096)
        blocks = 4096;
    hipLaunchKernelGGL(dgrad_weight_transform_kernel, dim3((unsigned)blocks), dim3(256), 0, s, W,
                       Wt, G, Kg, Cg, kh, kw, sh, sw, Th, Tw, tk);
    return hipGetLastError();
}

// Fixed-order sums: out[i] = (acc ? out[i] : 0) + sum_s P[s][i],
// db[k] = (acc ? db[k] : 0) + sum_n sums[n*K + k].
// A block owns 32 consecutive outputs; its 8 waves-of-32-lanes each add the
// terms q = part, part + 8, ... in order (lanes along i: coalesced), then one
// lane per output adds the 8 part sums in order.  The association is fixed
// by (count of terms, 8), so results are bitwise reproducible.
constexpr int kRedParts = 8;
constexpr int kRedCols = 32;

__global__ void __launch_bounds__(kRedParts * kRedCols)
wgrad_reduce_kernel(const float* __restrict__ P, float* __restrict__ out, int count, int splits,
                    const float* __restrict__ plane_sums, float* __restrict__ db, int N, int K,
                    int accumulate)
{
    __shared__ float part[kRedParts][kRedCols + 1];
    const int col = threadIdx.x % kRedCols;
    const int pt = threadIdx.x / kRedCols;
    const int e = blockIdx.x * kRedCols + col;
    const int total = count + (db ? K : 0);
    const bool is_w = e < count;
    const float* src = is_w ? P + e : plane_sums + (e - count);
    const size_t stride = is_w ? (size_t)count : (size_t)K;
    const int terms = is_w ? splits : N;
    float s = 0.f;
    if (e < total) {
        int q = pt;
        for (; q + 3 * kRedParts < terms; q += 4 * kRedParts) {
            const float a0 = src[(size_t)q * stride];
            const float a1 = src[(size_t)(q + kRedParts) * stride];
            const float a2 = src[(size_t)(q + 2 * kRedParts) * stride];
            const float a3 = src[(size_t)(q + 3 * kRedParts) * stride];
            s += a0;
            s += a1;
            s += a2;
            s += a3;
        }
        for (; q < terms; q += kRedParts)
            s += src[(size_t)q * stride];
    }
    part[pt][col] = s;
    __syncthreads();
    if (pt == 0 && e < total) {
        float t = 0.f;
#pragma unroll
        for (int i = 0; i < kRedParts; ++i)
            t += part[i][col];
        if (is_w)
            out[e] = accumulate ? out[e] + t : t;
        else
            db[e - count] = accumulate ? db[e - count] + t : t;
    }
}

hipError_t launch_wgrad_reduce(const float* P, float* out, int count, int splits,
                               const float* plane_sums, float* db, int N, int K, int accumulate,
                               hipStream_t s)
{
    const int total = count + (db ? K : 0);
    if (total == 0)
        return hipSuccess;
    const int blocks = (total + kRedCols - 1) / kRedCols;
    hipLaunchKernelGGL(wgrad_reduce_kernel, dim3(blocks), dim3(kRedParts * kRedCols), 0, s, P, out,
                       count, splits, plane_sums, db, N, K, accumulate);
    return hipGetLastError();
}

// 32 x 32 tiles through LDS: coalesced reads along c, coalesced writes along r.
__global__ void __launch_bounds__(256)
transpose_f32_kernel(const float* __restrict__ in, float* __restrict__ out, int R, int C)
{
    __shared__ float tile[32][33];
    const int c0 = blockIdx.x * 32, r0 = blockIdx.y * 32;
    const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
#pragma unroll
    for (int k = 0; k < 32; k += 8) {
        const int r = r0 + ty + k, c = c0 + tx;
        if (r < R && c < C)
            tile[ty + k][tx] = in[(size_t)r * C + c];
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 32; k += 8) {
        const int c = c0 + ty + k, r = r0 + tx;
        if (r < R && c < C)
            out[(size_t)c * R + r] = tile[tx][ty + k];
    }
}

hipError_t launch_transpose_f32(const float* in, float* out, int R, int C, hipStream_t s)
{
    if ((long)R * C == 0)
        return hipSuccess;
    hipLaunchKernelGGL(transpose_f32_kernel, dim3((C + 31) / 32, (R + 31) / 32), dim3(256), 0, s,
                       in, out, R, C);
    return hipGetLastError();
}

// Split-K partials added in order (s = 0, 1, ...), then the bias and ReLU.
__global__ void __launch_bounds__(256)
split_reduce_kernel(const float* __restrict__ P, int splits, int count, int ncol,
                    const float* __restrict__ bias, int relu, const float* __restrict__ mask,
                    float* __restrict__ out)
{
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < count;
         i += gridDim.x * blockDim.x) {
        float t = 0.f;
        for (int q = 0; q < splits; ++q)
            t += P[(size_t)q * count + i];
        if (bias)
            t += bias[i % ncol];
        if (relu && !(t > 0.f))
            t = 0.f;
        if (mask && !(mask[i] > 0.f))
            t = 0.f;
        out[i] = t;
    }
}

hipError_t launch_split_reduce(const float* P, int splits, int count, int ncol, const float* bias,
                               int relu, const float* mask, float* out, hipStream_t s)
{
    if (count == 0)
        return hipSuccess;
    int blocks = (count + 255) / 256;
    if (blocks > 8192)
        blocks = 8192;
    hipLaunchKernelGGL(split_reduce_kernel, dim3(blocks), dim3(256), 0, s, P, splits, count, ncol,
                       bias, relu, mask, out);
    return hipGetLastError();
}

// Split convolution GEMM epilogues: one thread per GEMM output (g, m, col),
// col fastest (coalesced partial reads); the partials of an output are added
// in split order after the bias.
// The region: groups g0 .. g0 + Gt - 1, columns c0 .. c0 + Nc - 1.
__global__ void __launch_bounds__(256)
conv_split_reduce_fwd_kernel(const float* __restrict__ P, int splits, int g0, int Gt, int M,
                             int c0, int Nc, int OHW, int Cout, const float* __restrict__ bias,
                             int relu, float* __restrict__ Y)
{
    const int64_t count = (int64_t)Gt * M * Nc;
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < count;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int col = c0 + (int)(e % Nc);
        const int gm = g0 * M + (int)(e / Nc);     // g * M + m = output channel
        float t = bias ? bias[gm] : 0.f;
        for (int q = 0; q < splits; ++q)
            t += P[(int64_t)q * count + e];
        const int n = col / OHW;
        const int pix = col - n * OHW;
        Y[((int64_t)n * Cout + gm) * OHW + pix] = t > 0.f ? t : (relu ? 0.f : t);
    }
}

__global__ void __launch_bounds__(256)
conv_split_reduce_dgrad_kernel(const float* __restrict__ P, int splits, int g0, int Gt, int M,
                               int c0, int Nc, int OHW, int OW, int psh, int psw, int a0h,
                               int a0w, int oph, int opw, int Cout, int Cg_out, int OutH,
                               int OutW, const float* __restrict__ mask, float* __restrict__ dX)
{
    const int64_t count = (int64_t)Gt * M * Nc;
    const int pss = psh * psw;
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < count;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int col = c0 + (int)(e % Nc);
        const int gm = g0 * M + (int)(e / Nc);
        const int g = gm / M;
        const int m = gm - g * M;
        const int c = m / pss;
        const int fr = m - c * pss;
        const int fh = fr / psw;
        const int fw = fr - fh * psw;
        const int n = col / OHW;
        const int pix = col - n * OHW;
        const int a = pix / OW;
        const int b = pix - a * OW;
        const int h = psh * (a + a0h) - oph + fh;
        const int w = psw * (b + a0w) - opw + fw;
        if ((unsigned)h >= (unsigned)OutH || (unsigned)w >= (unsigned)OutW)
            continue;
        float t = 0.f;
        for (int q = 0; q < splits; ++q)
            t += P[(int64_t)q * count + e];
        const int64_t o = (((int64_t)n * Cout + g * Cg_out + c) * OutH + h) * OutW + w;
        if (mask && !(mask[o] > 0.f))
            t = 0.f;
        dX[o] = t;
    }
}

hipError_t launch_conv_split_reduce_fwd(const float* P, int splits, const ConvGemmParams& q,
                                        float* Y, hipStream_t s, int g0, int c0)
{
    if (g0 < 0 || g0 > q.G || c0 < 0 || c0 > q.Ncol)
        return hipErrorInvalidValue;
    const int Gt = q.G - g0, Nc = q.Ncol - c0;
    const int64_t count = (int64_t)Gt * q.M * Nc;
    if (count == 0)
        return hipSuccess;
    int64_t blocks = (count + 255) / 256;
    if (blocks > 8192)
        blocks = 8192;
    hipLaunchKernelGGL(conv_split_reduce_fwd_kernel, dim3((unsigned)blocks), dim3(256), 0, s, P,
                       splits, g0, Gt, q.M, c0, Nc, q.OH * q.OW, q.Cout, q.bias, q.relu, Y);
    return hipGetLastError();
}

hipError_t launch_conv_split_reduce_dgrad(const float* P, int splits, const ConvGemmParams& q,
                                          const float* mask, float* dX, hipStream_t s, int g0,
                                          int c0)
{
    if (g0 < 0 || g0 > q.G || c0 < 0 || c0 > q.Ncol)
        return hipErrorInvalidValue;
    const int Gt = q.G - g0, Nc = q.Ncol - c0;
    const int64_t count = (int64_t)Gt * q.M * Nc;
    if (count == 0)
        return hipSuccess;
    int64_t blocks = (count + 255) / 256;
    if (blocks > 8192)
        blocks = 8192;
    hipLaunchKernelGGL(conv_split_reduce_dgrad_kernel, dim3((unsigned)blocks), dim3(256), 0, s, P,
                       splits, g0, Gt, q.M, c0, Nc, q.OH * q.OW, q.OW, q.psh, q.psw, q.a0h,
                       q.a0w, q.oph, q.opw, q.Cout, q.Cg_out, q.OutH, q.OutW, mask, dX);
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
