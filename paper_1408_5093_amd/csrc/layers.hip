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
// Grid: x over 256-pixel tiles of a plane, y over planes (n, c); pixel
// coordinates come from a multiply-shift division.  KS/SS fix the window and
// stride at compile time (0 = runtime).
__device__ __forceinline__ int udiv(int x, const FastDiv& f)
{
    return (int)(((uint64_t)(uint32_t)x * f.mul) >> f.shift);
}

// Each thread owns PPT planes at the same pixel (planes nc, nc + NCg, ...):
// all their loads are independent, which keeps enough memory traffic in
// flight for these short, latency-bound kernels.
constexpr int kPoolPlanesPerThread = 4;

template <int KS, int SS>
__global__ void __launch_bounds__(256)
maxpool_forward_kernel(const float* __restrict__ x, float* __restrict__ y,
                       int32_t* __restrict__ mask, int NC, int H, int W, int OH, int OW, int kh_,
                       int kw_, int sh_, int sw_, int ph, int pw, FastDiv div_ow, int relu_input,
                       int mask_u8)
{
    constexpr int PPT = kPoolPlanesPerThread;
    const int kh = KS ? KS : kh_, kw = KS ? KS : kw_;
    const int sh = SS ? SS : sh_, sw = SS ? SS : sw_;
    const int OHW = OH * OW;
    const int p = blockIdx.x * 256 + threadIdx.x;
    if (p >= OHW)
        return;
    const int i = udiv(p, div_ow);
    const int j = p - i * OW;
    const int hs = i * sh - ph, ws = j * sw - pw;
    const int h0 = max(hs, 0), w0 = max(ws, 0);
    const int first = h0 * W + w0;
    const int stride = gridDim.y;  // planes handled by one grid row
    for (int nc0 = blockIdx.y; nc0 < NC; nc0 += stride * PPT) {
        float bv[PPT];
        int best[PPT], boff[PPT];  // the winner: plane index, offset in the window
        if constexpr (KS > 0) {
            // fixed window: every load is independent; out-of-image taps are
            // replaced by the window's first tap (strict '>' keeps the first
            // maximum in row-major order)
            float v[PPT][KS][KS];
#pragma unroll
            for (int t = 0; t < PPT; ++t) {
                const int nc = min(nc0 + t * stride, NC - 1);
                const float* plane = x + nc * (H * W);
                bv[t] = plane[first];
#pragma unroll
                for (int du = 0; du < KS; ++du)
#pragma unroll
                    for (int dv = 0; dv < KS; ++dv) {
                        const int h = hs + du, w = ws + dv;
                        const bool in = (unsigned)h < (unsigned)H && (unsigned)w < (unsigned)W;
                        v[t][du][dv] = plane[in ? h * W + w : first];
                    }
            }
#pragma unroll
            for (int t = 0; t < PPT; ++t) {
                best[t] = first;
                boff[t] = (h0 - hs) * KS + (w0 - ws);
#pragma unroll
                for (int du = 0; du < KS; ++du)
#pragma unroll
                    for (int dv = 0; dv < KS; ++dv)
                        if (v[t][du][dv] > bv[t]) {
                            bv[t] = v[t][du][dv];
                            best[t] = (hs + du) * W + ws + dv;
                            boff[t] = du * KS + dv;
                        }
            }
        } else {
            const int h1 = min(hs + kh, H), w1 = min(ws + kw, W);
#pragma unroll
            for (int t = 0; t < PPT; ++t) {
                const int nc = min(nc0 + t * stride, NC - 1);
                const float* plane = x + nc * (H * W);
                bv[t] = plane[first];
                best[t] = first;
                boff[t] = (h0 - hs) * kw + (w0 - ws);
                for (int h = h0; h < h1; ++h)
                    for (int w = w0; w < w1; ++w) {
                        const float v = plane[h * W + w];
                        if (v > bv[t]) {
                            bv[t] = v;
                            best[t] = h * W + w;
                            boff[t] = (h - hs) * kw + (w - ws);
                        }
                    }
            }
        }
#pragma unroll
        for (int t = 0; t < PPT; ++t) {
            const int nc = nc0 + t * stride;
            if (nc < NC) {
                y[nc * OHW + p] = bv[t];
                // a ReLU output window with no positive value routes nothing
                const bool none = relu_input && !(bv[t] > 0.f);
                if (mask && mask_u8)
                    ((uint8_t*)mask)[nc * OHW + p] = none ? (uint8_t)255 : (uint8_t)boff[t];
                else if (mask)
                    mask[nc * OHW + p] = none ? -1 : best[t];
            }
        }
    }
}

// Gather form (one thread per input position, covering outputs visited in
// row-major order): deterministic, no atomics.  With a fixed window, at most
// ceil(KS/SS)^2 outputs cover an input; their masks and gradients are loaded
// unconditionally (clamped indices), then added in order where the mask
// names this input.
template <int KS, int SS>
__global__ void __launch_bounds__(256)
maxpool_backward_kernel(const float* __restrict__ dy, const int32_t* __restrict__ mask,
                        float* __restrict__ dx, int NC, int H, int W, int OH, int OW, int kh_,
                        int kw_, int sh_, int sw_, int ph, int pw, FastDiv div_w)
{
    constexpr int PPT = kPoolPlanesPerThread;
    const int kh = KS ? KS : kh_, kw = KS ? KS : kw_;
    const int sh = SS ? SS : sh_, sw = SS ? SS : sw_;
    const int HW = H * W;
    const int p = blockIdx.x * 256 + threadIdx.x;
    if (p >= HW)
        return;
    const int h = udiv(p, div_w);
    const int w = p - h * W;
    // outputs whose window covers (h, w): i*sh - ph <= h <= i*sh - ph + kh - 1
    const int i0 = max(0, (h + ph - kh + sh) / sh);
    const int i1 = min(OH - 1, (h + ph) / sh);
    const int j0 = max(0, (w + pw - kw + sw) / sw);
    const int j1 = min(OW - 1, (w + pw) / sw);
    const int stride = gridDim.y;
    for (int nc0 = blockIdx.y; nc0 < NC; nc0 += stride * PPT) {
        float s[PPT];
        if constexpr (KS > 0) {
            constexpr int T = (KS + SS - 1) / SS;
            int mk[PPT][T][T];
            float g[PPT][T][T];
#pragma unroll
            for (int t = 0; t < PPT; ++t) {
                const int obase = min(nc0 + t * stride, NC - 1) * (OH * OW);
#pragma unroll
                for (int di = 0; di < T; ++di)
#pragma unroll
                    for (int dj = 0; dj < T; ++dj) {
                        const int o = obase + min(i0 + di, OH - 1) * OW + min(j0 + dj, OW - 1);
                        mk[t][di][dj] = mask[o];
                        g[t][di][dj] = dy[o];
                    }
            }
#pragma unroll
            for (int t = 0; t < PPT; ++t) {
                s[t] = 0.f;
#pragma unroll
                for (int di = 0; di < T; ++di)
#pragma unroll
                    for (int dj = 0; dj < T; ++dj)
                        if (i0 + di <= i1 && j0 + dj <= j1 && mk[t][di][dj] == p)
                            s[t] += g[t][di][dj];
            }
        } else {
#pragma unroll
            for (int t = 0; t < PPT; ++t) {
                const int obase = min(nc0 + t * stride, NC - 1) * (OH * OW);
                s[t] = 0.f;
                for (int i = i0; i <= i1; ++i)
                    for (int j = j0; j <= j1; ++j)
                        if (mask[obase + i * OW + j] == p)
                            s[t] += dy[obase + i * OW + j];
            }
        }
#pragma unroll
        for (int t = 0; t < PPT; ++t) {
            const int nc = nc0 + t * stride;
            if (nc < NC)
                dx[nc * HW + p] = s[t];
        }
    }
}

// Plane-staged variants for planes that fit in LDS: a block copies PB whole
// consecutive planes (one contiguous run of memory) into LDS with coalesced
// loads, so every input is read from HBM once and the overlapping windows
// are served from LDS; outputs are written coalesced in plane order.
constexpr int kPoolLdsFloats = 8192;  // 32 KB of staged planes per block

template <int KS, int SS>
__global__ void __launch_bounds__(256)
maxpool_forward_lds_kernel(const float* __restrict__ x, float* __restrict__ y,
                           int32_t* __restrict__ mask, int NC, int H, int W, int OH, int OW,
                           int kh_, int kw_, int sh_, int sw_, int ph, int pw, int PB,
                           FastDiv div_ohw, FastDiv div_ow, int relu_input, int mask_u8)
{
    __shared__ float xs[kPoolLdsFloats];
    const int kh = KS ? KS : kh_, kw = KS ? KS : kw_;
    const int sh = SS ? SS : sh_, sw = SS ? SS : sw_;
    const int HW = H * W, OHW = OH * OW;
    const int nc0 = blockIdx.x * PB;
    const int np = min(PB, NC - nc0);
    const float* src = x + (size_t)nc0 * HW;
    const int ne = np * HW;
    // thirty-two independent loads in flight per thread (a whole block's
    // staging at once for planes of up to 8192 floats), then their LDS stores
    // (with sixteen, pool1 at N=256 ran 8% slower; with eight, ~4.4 TB/s)
    for (int e0 = threadIdx.x; e0 < ne; e0 += 256 * 32) {
        float v[32];
#pragma unroll
        for (int u = 0; u < 32; ++u)
            v[u] = e0 + 256 * u < ne ? src[e0 + 256 * u] : 0.f;
#pragma unroll
        for (int u = 0; u < 32; ++u)
            if (e0 + 256 * u < ne)
                xs[e0 + 256 * u] = v[u];
    }
    __syncthreads();
    for (int o = threadIdx.x; o < np * OHW; o += 256) {
        const int pl = udiv(o, div_ohw);
        const int p = o - pl * OHW;
        const int i = udiv(p, div_ow);
        const int j = p - i * OW;
        const int hs = i * sh - ph, ws = j * sw - pw;
        const int h0 = max(hs, 0), w0 = max(ws, 0);
        const int h1 = min(hs + kh, H), w1 = min(ws + kw, W);
        const float* plane = xs + pl * HW;
        const int first = h0 * W + w0;
        float bv = plane[first];
        int best = first;
        int boff = (h0 - hs) * kw + (w0 - ws);  // the winner's offset in its window
        if constexpr (KS > 0) {
            // all taps read first; taps outside the image read the window's
            // first tap, which never wins the strict '>' below
            float v[KS][KS];
#pragma unroll
            for (int du = 0; du < KS; ++du)
#pragma unroll
                for (int dv = 0; dv < KS; ++dv) {
                    const int h = hs + du, w = ws + dv;
                    const bool in = (unsigned)h < (unsigned)H && (unsigned)w < (unsigned)W;
                    v[du][dv] = plane[in ? h * W + w : first];
                }
#pragma unroll
            for (int du = 0; du < KS; ++du)
#pragma unroll
                for (int dv = 0; dv < KS; ++dv)
                    if (v[du][dv] > bv) {
                        bv = v[du][dv];
                        best = (hs + du) * W + ws + dv;
                        boff = du * KS + dv;
                    }
        } else {
            for (int h = h0; h < h1; ++h)
                for (int w = w0; w < w1; ++w) {
                    const float v = plane[h * W + w];
                    if (v > bv) {
                        bv = v;
                        best = h * W + w;
                        boff = (h - hs) * kw + (w - ws);
                    }
                }
        }
        const size_t out = (size_t)nc0 * OHW + o;
        y[out] = bv;
        // a ReLU output window with no positive value routes nothing
        const bool none = relu_input && !(bv > 0.f);
        if (mask && mask_u8)
            ((uint8_t*)mask)[out] = none ? (uint8_t)255 : (uint8_t)boff;
        else if (mask)
            mask[out] = none ? -1 : best;
    }
}

// Gather form from staged masks and gradients: each input position adds, in
// row-major output order, the gradients of the covering windows whose mask
// names it.
template <int KS, int SS>
__global__ void __launch_bounds__(256)
maxpool_backward_lds_kernel(const float* __restrict__ dy, const int32_t* __restrict__ mask,
                            float* __restrict__ dx, int NC, int H, int W, int OH, int OW, int kh_,
                            int kw_, int sh_, int sw_, int ph, int pw, int PB, FastDiv div_hw,
                            FastDiv div_w)
{
    __shared__ float gs[kPoolLdsFloats / 2];
    __shared__ int32_t ms[kPoolLdsFloats / 2];
    const int kh = KS ? KS : kh_, kw = KS ? KS : kw_;
    const int sh = SS ? SS : sh_, sw = SS ? SS : sw_;
    const int HW = H * W, OHW = OH * OW;
    const int nc0 = blockIdx.x * PB;
    const int np = min(PB, NC - nc0);
    const size_t obase = (size_t)nc0 * OHW;
    const int ne = np * OHW;
    for (int e0 = threadIdx.x; e0 < ne; e0 += 256 * 4) {
        float g[4];
        int32_t m[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const bool in = e0 + 256 * u < ne;
            g[u] = in ? dy[obase + e0 + 256 * u] : 0.f;
            m[u] = in ? mask[obase + e0 + 256 * u] : -1;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u)
            if (e0 + 256 * u < ne) {
                gs[e0 + 256 * u] = g[u];
                ms[e0 + 256 * u] = m[u];
            }
    }
    __syncthreads();
    for (int e = threadIdx.x; e < np * HW; e += 256) {
        const int pl = udiv(e, div_hw);
        const int p = e - pl * HW;
        const int h = udiv(p, div_w);
        const int w = p - h * W;
        const int i0 = max(0, (h + ph - kh + sh) / sh);
        const int i1 = min(OH - 1, (h + ph) / sh);
        const int j0 = max(0, (w + pw - kw + sw) / sw);
        const int j1 = min(OW - 1, (w + pw) / sw);
        const int ob = pl * OHW;
        float sum = 0.f;
        if constexpr (KS > 0) {
            // covering windows read first (indices clamped into the plane),
            // then added in row-major order where valid and routed here
            constexpr int T = (KS + SS - 1) / SS;
            int m[T][T];
            float g[T][T];
#pragma unroll
            for (int di = 0; di < T; ++di)
#pragma unroll
                for (int dj = 0; dj < T; ++dj) {
                    const int o = ob + min(i0 + di, OH - 1) * OW + min(j0 + dj, OW - 1);
                    m[di][dj] = ms[o];
                    g[di][dj] = gs[o];
                }
#pragma unroll
            for (int di = 0; di < T; ++di)
#pragma unroll
                for (int dj = 0; dj < T; ++dj)
                    if (i0 + di <= i1 && j0 + dj <= j1 && m[di][dj] == p)
                        sum += g[di][dj];
        } else {
            for (int i = i0; i <= i1; ++i)
                for (int j = j0; j <= j1; ++j) {
                    const int o = ob + i * OW + j;
                    if (ms[o] == p)
                        sum += gs[o];
                }
        }
        dx[(size_t)nc0 * HW + e] = sum;
    }
}

static unsigned grid_for(long total)
{
    long b = (total + 255) / 256;
    return (unsigned)(b > 16384 ? 16384 : (b < 1 ? 1 : b));
}

static unsigned grid_exact(long total) { return (unsigned)((total + 255) / 256); }

static dim3 plane_grid(int pixels, int planes)
{
    // y covers the planes kPoolPlanesPerThread at a time
    const int rows = (planes + kPoolPlanesPerThread - 1) / kPoolPlanesPerThread;
    return dim3((unsigned)((pixels + 255) / 256), (unsigned)(rows < 65535 ? rows : 65535));
}

hipError_t launch_maxpool_forward(const float* x, float* y, int32_t* mask, int NC, int H, int W,
                                  int OH, int OW, int kh, int kw, int sh, int sw, int ph, int pw,
                                  int relu_input, hipStream_t s, int mask_u8)
{
    if ((long)NC * OH * OW == 0)
        return hipSuccess;
    if (mask_u8 && kh * kw > 255)
        return hipErrorInvalidValue;
    const FastDiv d = make_fastdiv((uint32_t)OW);
    if (H * W <= kPoolLdsFloats) {
        // planes staged in LDS, as many whole planes per block as fit
        const int PB = kPoolLdsFloats / (H * W);
        const dim3 g((unsigned)((NC + PB - 1) / PB));
        const FastDiv dohw = make_fastdiv((uint32_t)(OH * OW));
        if (kh == 3 && kw == 3 && sh == 2 && sw == 2)
            hipLaunchKernelGGL((maxpool_forward_lds_kernel<3, 2>), g, dim3(256), 0, s, x, y, mask,
                               NC, H, W, OH, OW, kh, kw, sh, sw, ph, pw, PB, dohw, d, relu_input,
                               mask_u8);
        else if (kh == 2 && kw == 2 && sh == 2 && sw == 2)
            hipLaunchKernelGGL((maxpool_forward_lds_kernel<2, 2>), g, dim3(256), 0, s, x, y, mask,
                               NC, H, W, OH, OW, kh, kw, sh, sw, ph, pw, PB, dohw, d, relu_input,
                               mask_u8);
        else
            hipLaunchKernelGGL((maxpool_forward_lds_kernel<0, 0>), g, dim3(256), 0, s, x, y, mask,
                               NC, H, W, OH, OW, kh, kw, sh, sw, ph, pw, PB, dohw, d, relu_input,
                               mask_u8);
        return hipGetLastError();
    }
    const dim3 grid = plane_grid(OH * OW, NC);
    if (kh == 3 && kw == 3 && sh == 2 && sw == 2)
        hipLaunchKernelGGL((maxpool_forward_kernel<3, 2>), grid, dim3(256), 0, s, x, y, mask, NC,
                           H, W, OH, OW, kh, kw, sh, sw, ph, pw, d, relu_input, mask_u8);
    else if (kh == 2 && kw == 2 && sh == 2 && sw == 2)
        hipLaunchKernelGGL((maxpool_forward_kernel<2, 2>), grid, dim3(256), 0, s, x, y, mask, NC,
                           H, W, OH, OW, kh, kw, sh, sw, ph, pw, d, relu_input, mask_u8);
    else
        hipLaunchKernelGGL((maxpool_forward_kernel<0, 0>), grid, dim3(256), 0, s, x, y, mask, NC,
                           H, W, OH, OW, kh, kw, sh, sw, ph, pw, d, relu_input, mask_u8);
    return hipGetLastError();
}

hipError_t launch_maxpool_backward(const float* dy, const int32_t* mask, float* dx, int NC, int H,
                                   int W, int OH, int OW, int kh, int kw, int sh, int sw, int ph,
                                   int pw, hipStream_t s)
{
    if ((long)NC * H * W == 0)
        return hipSuccess;
    const FastDiv d = make_fastdiv((uint32_t)W);
    if (OH * OW <= kPoolLdsFloats / 2) {
        const int PB = (kPoolLdsFloats / 2) / (OH * OW);
        const dim3 g((unsigned)((NC + PB - 1) / PB));
        const FastDiv dhw = make_fastdiv((uint32_t)(H * W));
        if (kh == 3 && kw == 3 && sh == 2 && sw == 2)
            hipLaunchKernelGGL((maxpool_backward_lds_kernel<3, 2>), g, dim3(256), 0, s, dy, mask,
                               dx, NC, H, W, OH, OW, kh, kw, sh, sw, ph, pw, PB, dhw, d);
        else if (kh == 2 && kw == 2 && sh == 2 && sw == 2)
            hipLaunchKernelGGL((maxpool_backward_lds_kernel<2, 2>), g, dim3(256), 0, s, dy, mask,
                               dx, NC, H, W, OH, OW, kh, kw, sh, sw, ph, pw, PB, dhw, d);
        else
            hipLaunchKernelGGL((maxpool_backward_lds_kernel<0, 0>), g, dim3(256), 0, s, dy, mask,
                               dx, NC, H, W, OH, OW, kh, kw, sh, sw, ph, pw, PB, dhw, d);
        return hipGetLastError();
    }
    const dim3 grid = plane_grid(H * W, NC);
    if (kh == 3 && kw == 3 && sh == 2 && sw == 2)
        hipLaunchKernelGGL((maxpool_backward_kernel<3, 2>), grid, dim3(256), 0, s, dy, mask, dx,
                           NC, H, W, OH, OW, kh, kw, sh, sw, ph, pw, d);
    else if (kh == 2 && kw == 2 && sh == 2 && sw == 2)
        hipLaunchKernelGGL((maxpool_backward_kernel<2, 2>), grid, dim3(256), 0, s, dy, mask, dx,
                           NC, H, W, OH, OW, kh, kw, sh, sw, ph, pw, d);
    else
        hipLaunchKernelGGL((maxpool_backward_kernel<0, 0>), grid, dim3(256), 0, s, dy, mask, dx,
                           NC, H, W, OH, OW, kh, kw, sh, sw, ph, pw, d);
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
__device__ __forceinline__ float pow_neg(float s, float beta)
{
    // s^-beta for s >= k > 0 via the hardware exp2/log2 (about 1 ulp each)
    return __builtin_amdgcn_exp2f(-beta * __builtin_amdgcn_logf(s));
}

// The output's bf16 staging for a convolution that takes it as its bottom
// (LrnStage): Xp[n][h + tb][w + lb][c] on an Hp x Wp grid of C channels.
// Work mapping of the staging variant: a wave takes 64 pixels of one
// chunk; a block, `wpb` chunks of the same 64 pixels; the `nb` blocks of a
// pixel group (image n, pixels 64 grp ..) sit 8 ids apart, so that they run
// on one XCD and each staged pixel's channels are written through one L2.
struct LrnStage {
    uint16_t* Xp;
    int W, Hp, Wp, tb, lb;
    int npg, nb, wpb;  // pixel groups per image, blocks per group, waves per block
};

// One thread per (n, chunk of CH channels, pixel); lanes run along pixels.
// Every input of the chunk and its halo is loaded up front (independent
// loads), then the outputs are formed from registers.  STAGE: the chunk's
// outputs also go to the staging, rounded to bf16 (two 16-byte stores).
template <int SIZE, int CH, bool STAGE = false>
__global__ void __launch_bounds__(256)
lrn_forward_kernel(const float* __restrict__ x, float* __restrict__ y, int N, int C, int HW,
                   int nchunks, FastDiv div_hw, float alpha_over_n, float beta, float k,
                   LrnStage st = LrnStage{})
{
    constexpr int PRE = (SIZE - 1) / 2;
    constexpr int NA = CH + SIZE - 1;
    int n, c0, pix;
    if constexpr (STAGE) {
        const int xcd = blockIdx.x & 7;
        const int r = blockIdx.x >> 3;
        const int j = r % st.nb;
        const int pg = (r / st.nb) * 8 + xcd;
        if (pg >= N * st.npg)
            return;
        n = pg / st.npg;
        pix = (pg - n * st.npg) * 64 + (threadIdx.x & 63);
        c0 = (j * st.wpb + (threadIdx.x >> 6)) * CH;
        if (pix >= HW)
            return;
    } else {
        const int e = blockIdx.x * blockDim.x + threadIdx.x;
        if (e >= N * nchunks * HW)
            return;
        const int rest = udiv(e, div_hw);
        pix = e - rest * HW;
        n = rest / nchunks;
        c0 = (rest - n * nchunks) * CH;
    }
    // Range-checked buffer accesses: a channel outside [0, C) gets an offset
    // with bit 31 set, which reads 0 / drops the store, so every load is
    // unconditional and all of them are in flight together.
    const uint32_t bytes = (uint32_t)(N * C * HW) * 4u;
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(x, bytes);
    // (staging without y: an empty range, every store of y dropped)
    const __amdgpu_buffer_rsrc_t ry = make_rsrc(y, y ? bytes : 0u);
    const uint32_t base4 = (uint32_t)(n * C * HW + pix) * 4u;
    const uint32_t hw4 = (uint32_t)HW * 4u;
    auto off = [&](int ch) {
        return (base4 + (uint32_t)ch * hw4) | ((uint32_t)((unsigned)ch >= (unsigned)C) << 31);
    };
    float a[NA];  // channels c0 - PRE .. c0 + CH - 1 + POST
#pragma unroll
    for (int q = 0; q < NA; ++q)
        a[q] = buf_ld_f32(rx, off(c0 - PRE + q));
    uint32_t packed[CH / 2];
    float even = 0.f;
#pragma unroll
    for (int t = 0; t < CH; ++t) {
        // explicit fused multiply-adds: every instantiation rounds alike
        float sq = 0.f;
#pragma unroll
        for (int q = 0; q < SIZE; ++q)
            sq = __builtin_fmaf(a[t + q], a[t + q], sq);
        const float out = a[t + PRE] * pow_neg(__builtin_fmaf(alpha_over_n, sq, k), beta);
        buf_st_f32(out, ry, off(c0 + t));
        if constexpr (STAGE) {
            if (t & 1)
                packed[t >> 1] = f32x2_to_bf16x2_rne(even, out);
            else
                even = out;
        }
    }
    if constexpr (STAGE) {
        static_assert(CH % 8 == 0, "whole 16-byte chunks");
        // (C is a multiple of CH: the chunk lies inside the image's channels)
        const int h = pix / st.W;
        const int w = pix - h * st.W;
        uint16_t* dst =
            st.Xp + (((size_t)n * st.Hp + h + st.tb) * st.Wp + w + st.lb) * C + c0;
#pragma unroll
        for (int j = 0; j < CH / 8; ++j)
            *(u32x4*)(dst + 8 * j) = u32x4{packed[4 * j], packed[4 * j + 1], packed[4 * j + 2],
                                           packed[4 * j + 3]};
    }
}

// dx_c = g_c s_c^-beta - (2 alpha beta / size) a_c sum_{c' in [c - POST, c + PRE]} g_c' b_c' / s_c'
template <int SIZE, int CH>
__global__ void __launch_bounds__(256)
lrn_backward_kernel(const float* __restrict__ x, const float* __restrict__ y,
                    const float* __restrict__ dy, float* __restrict__ dx, int N, int C, int HW,
                    int nchunks, FastDiv div_hw, float alpha_over_n, float beta, float k)
{
    constexpr int PRE = (SIZE - 1) / 2;
    constexpr int POST = SIZE - 1 - PRE;
    constexpr int NR = CH + SIZE - 1;      // ratios: channels c0 - POST .. c0 + CH - 1 + PRE
    constexpr int NA = NR + SIZE - 1;      // inputs: channels c0 - POST - PRE .. + NA - 1
    const int e = blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= N * nchunks * HW)
        return;
    const int rest = udiv(e, div_hw);
    const int pix = e - rest * HW;
    const int n = rest / nchunks;
    const int c0 = (rest - n * nchunks) * CH;
    // range-checked buffer accesses, as in the forward kernel
    const uint32_t bytes = (uint32_t)(N * C * HW) * 4u;
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(x, bytes);
    const __amdgpu_buffer_rsrc_t ry = make_rsrc(y, bytes);
    const __amdgpu_buffer_rsrc_t rg = make_rsrc(dy, bytes);
    const __amdgpu_buffer_rsrc_t rd = make_rsrc(dx, bytes);
    const uint32_t base4 = (uint32_t)(n * C * HW + pix) * 4u;
    const uint32_t hw4 = (uint32_t)HW * 4u;
    auto off = [&](int ch) {
        return (base4 + (uint32_t)ch * hw4) | ((uint32_t)((unsigned)ch >= (unsigned)C) << 31);
    };
    float a[NA], g[NR], b[NR];
#pragma unroll
    for (int q = 0; q < NA; ++q)
        a[q] = buf_ld_f32(rx, off(c0 - POST - PRE + q));
#pragma unroll
    for (int q = 0; q < NR; ++q) {
        g[q] = buf_ld_f32(rg, off(c0 - POST + q));
        b[q] = buf_ld_f32(ry, off(c0 - POST + q));
    }
    float r[NR], sc[CH];
#pragma unroll
    for (int q = 0; q < NR; ++q) {
        float sq = 0.f;
#pragma unroll
        for (int t = 0; t < SIZE; ++t)
            sq += a[q + t] * a[q + t];
        const float s = k + alpha_over_n * sq;
        // hardware reciprocal (about 1 ulp): s >= k > 0
        r[q] = g[q] * b[q] * __builtin_amdgcn_rcpf(s);
        if (q >= POST && q < POST + CH)
            sc[q - POST] = s;
    }
    const float coef = 2.f * alpha_over_n * beta;
#pragma unroll
    for (int t = 0; t < CH; ++t) {
        float cross = 0.f;
#pragma unroll
        for (int q = 0; q < SIZE; ++q)
            cross += r[t + q];
        buf_st_f32(g[t + POST] * pow_neg(sc[t], beta) - coef * a[t + POST + PRE] * cross, rd,
                   off(c0 + t));
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

constexpr int kLrnChunk = 16;

hipError_t launch_lrn_forward(const float* x, float* y, int N, int C, int HW, int size,
                              float alpha, float beta, float k, hipStream_t s)
{
    if ((long)N * C * HW == 0)
        return hipSuccess;
    const float an = alpha / size;
    const int nch = (C + kLrnChunk - 1) / kLrnChunk;
    const long threads = (long)N * nch * HW;
    const FastDiv d = make_fastdiv((uint32_t)HW);
    if (size == 5)
        hipLaunchKernelGGL((lrn_forward_kernel<5, kLrnChunk>), dim3(grid_exact(threads)),
                           dim3(256), 0, s, x, y, N, C, HW, nch, d, an, beta, k);
    else if (size == 3)
        hipLaunchKernelGGL((lrn_forward_kernel<3, kLrnChunk>), dim3(grid_exact(threads)),
                           dim3(256), 0, s, x, y, N, C, HW, nch, d, an, beta, k);
    else
        hipLaunchKernelGGL(lrn_forward_any_kernel, dim3(grid_exact((long)N * C * HW)), dim3(256),
                           0, s, x, y, N, C, HW, size, an, beta, k);
    return hipGetLastError();
}

hipError_t launch_lrn_forward_stage(const float* x, float* y, int N, int C, int H, int W,
                                    int size, float alpha, float beta, float k, uint16_t* Xp,
                                    int Hp, int Wp, int tb, int lb, hipStream_t s)
{
    if ((long)N * C * H * W == 0)
        return hipSuccess;
    if (C % kLrnChunk != 0 || (size != 5 && size != 3) || tb < 0 || lb < 0 || Hp < tb + H ||
        Wp < lb + W || (((uintptr_t)Xp) & 15) != 0)
        return hipErrorInvalidValue;
    const hipError_t e = launch_dh_zero_border(Xp, N, Hp, Wp, tb, lb, H, W, C, s);
    if (e != hipSuccess)
        return e;
    const int HW = H * W;
    const float an = alpha / size;
    const int nch = C / kLrnChunk;
    const FastDiv d = make_fastdiv((uint32_t)HW);
    // waves per block: the largest divisor of the chunk count up to 4
    int wpb = 4;
    while (nch % wpb != 0)
        --wpb;
    const int npg = (HW + 63) / 64;
    const int nb = nch / wpb;
    const long groups8 = ((long)N * npg + 7) / 8;
    if (groups8 * 8 * nb > INT_MAX)
        return hipErrorInvalidValue;
    const LrnStage st{Xp, W, Hp, Wp, tb, lb, npg, nb, wpb};
    const dim3 grid((unsigned)(groups8 * 8 * nb)), block(64 * wpb);
    if (size == 5)
        hipLaunchKernelGGL((lrn_forward_kernel<5, kLrnChunk, true>), grid, block, 0, s, x, y, N, C,
                           HW, nch, d, an, beta, k, st);
    else
        hipLaunchKernelGGL((lrn_forward_kernel<3, kLrnChunk, true>), grid, block, 0, s, x, y, N, C,
                           HW, nch, d, an, beta, k, st);
    return hipGetLastError();
}

hipError_t launch_lrn_backward(const float* x, const float* y, const float* dy, float* dx, int N,
                               int C, int HW, int size, float alpha, float beta, float k,
                               hipStream_t s)
{
    if ((long)N * C * HW == 0)
        return hipSuccess;
    const float an = alpha / size;
    const int nch = (C + kLrnChunk - 1) / kLrnChunk;
    const long threads = (long)N * nch * HW;
    const FastDiv d = make_fastdiv((uint32_t)HW);
    if (size == 5)
        hipLaunchKernelGGL((lrn_backward_kernel<5, kLrnChunk>), dim3(grid_exact(threads)),
                           dim3(256), 0, s, x, y, dy, dx, N, C, HW, nch, d, an, beta, k);
    else if (size == 3)
        hipLaunchKernelGGL((lrn_backward_kernel<3, kLrnChunk>), dim3(grid_exact(threads)),
                           dim3(256), 0, s, x, y, dy, dx, N, C, HW, nch, d, an, beta, k);
    else
        hipLaunchKernelGGL(lrn_backward_any_kernel, dim3(grid_exact((long)N * C * HW)),
                           dim3(256), 0, s, x, y, dy, dx, N, C, HW, size, an, beta, k);
    return hipGetLastError();
}

// ------------------------------------------------------ fused LRN + max-pool backward
// The CaffeNet glue after conv1 and conv2 is max-pool then LRN over the pooled
// blob.  Its backward runs in one pass: a block owns (image, 16 channels, a
// strip of input rows); it forms the LRN backward (the pooled gradient) for
// every pooled row whose windows reach its input rows into LDS, then gathers
// each input position's gradient from LDS -- the pooled gradient never goes
// to HBM.  The arithmetic, and the order of every sum, is that of the
// separate LRN and pool kernels.  (The forward keeps the two separate
// kernels: the pooled blob must be stored for the backward anyway, so a
// one-pass forward saves only its re-read, and staging 20 channels of input
// rows per block left it slower than the plane-staged pool kernel.)
constexpr int kFuseCh = 16;      // channels owned by a block
constexpr int kFusePos = 256;    // pooled positions staged per block (one per thread)

// One block of the fused backward: image n, channels c0 .. c0 + 15, input
// rows y_lo .. y_hi, and the pooled rows i_lo .. i_hi whose windows reach
// them.
struct FuseBlock {
    int n, c0, strip, y_lo, y_hi, i_lo, i_hi;
};

__device__ __forceinline__ FuseBlock fuse_block(int H, int OH, int kh, int sh, int ph, int yrows,
                                                int nstrips, int nchunks)
{
    // Workgroups are dispatched round-robin over the 8 XCDs, each with its own
    // L2; neighbouring strips and channel chunks share halo rows and channels,
    // so each XCD takes one contiguous range of the block order.
    const int xcd = blockIdx.x & 7, per = gridDim.x >> 3, extra = gridDim.x & 7;
    const int blk = xcd * per + min(xcd, extra) + (blockIdx.x >> 3);
    FuseBlock f;
    f.strip = blk % nstrips;
    const int rest = blk / nstrips;
    f.c0 = (rest % nchunks) * kFuseCh;
    f.n = rest / nchunks;
    f.y_lo = f.strip * yrows;
    f.y_hi = min(H, f.y_lo + yrows) - 1;
    f.i_lo = max(0, (f.y_lo + ph - kh + sh) / sh);
    f.i_hi = min(OH - 1, (f.y_hi + ph) / sh);
    return f;
}

// Phase 1: the pooled gradient (LRN backward) of the block's 16 channels at
// every staged pooled position, and the winners, into LDS.
// The LRN's output b = a s^-beta is not read: it is formed again from the
// pooled inputs exactly as the forward kernel forms it (the same fused
// multiply-adds, the same hardware exp2 / log2), so it has the same bits,
// and the pass reads a fifth fewer bytes.
// With mask_u8 the mask holds each winner's offset du * kw + dv in its window
// (255: none), staged as the plane index it stands for.
template <int SIZE>
__device__ __forceinline__ void fuse_stage_pooled_grad(
    const FuseBlock& f, const float* __restrict__ a_in, const float* __restrict__ g_in,
    const int32_t* __restrict__ mask,
    float (&gs)[kFuseCh][kFusePos], int32_t (&ms)[kFuseCh][kFusePos], int N, int C, int OH, int OW,
    float alpha_over_n, float beta, float k, int mask_u8, int W, int kw, int sh, int sw, int ph,
    int pw)
{
    constexpr int PRE = (SIZE - 1) / 2;
    constexpr int POST = SIZE - 1 - PRE;
    constexpr int NR = kFuseCh + SIZE - 1;   // ratios: channels c0 - POST .. c0 + 15 + PRE
    constexpr int NA = NR + SIZE - 1;        // inputs: channels c0 - POST - PRE .. + NA - 1
    const int npos = (f.i_hi - f.i_lo + 1) * OW;
    const int OHW = OH * OW;
    const int c0 = f.c0;
    const int pos = threadIdx.x;
    if (pos >= npos)
        return;
    const int pi = f.i_lo + pos / OW, pj = pos - (pos / OW) * OW;
    const int pix = pi * OW + pj;
    const uint32_t bytes = (uint32_t)(N * C * OHW) * 4u;
    const __amdgpu_buffer_rsrc_t ra = make_rsrc(a_in, bytes);
    const __amdgpu_buffer_rsrc_t rg = make_rsrc(g_in, bytes);
    const __amdgpu_buffer_rsrc_t rm = make_rsrc(mask, mask_u8 ? bytes / 4u : bytes);
    const int wh0 = pi * sh - ph, ww0 = pj * sw - pw;  // the window's first position
    const uint32_t base4 = (uint32_t)(f.n * C * OHW + pix) * 4u;
    const uint32_t hw4 = (uint32_t)OHW * 4u;
    auto off = [&](int ch) {
        return (base4 + (uint32_t)ch * hw4) | ((uint32_t)((unsigned)ch >= (unsigned)C) << 31);
    };
    float a[NA], g[NR];
#pragma unroll
    for (int q = 0; q < NA; ++q)
        a[q] = buf_ld_f32(ra, off(c0 - POST - PRE + q));
#pragma unroll
    for (int q = 0; q < NR; ++q)
        g[q] = buf_ld_f32(rg, off(c0 - POST + q));
    float r[NR], pc[kFuseCh];
#pragma unroll
    for (int q = 0; q < NR; ++q) {
        // channel c0 - POST + q: its scale s, s^-beta and output b
        float sq = 0.f;
#pragma unroll
        for (int t = 0; t < SIZE; ++t)
            sq = __builtin_fmaf(a[q + t], a[q + t], sq);
        const float s = __builtin_fmaf(alpha_over_n, sq, k);
        const float p = pow_neg(s, beta);
        const float b = a[q + PRE] * p;
        r[q] = g[q] * b * __builtin_amdgcn_rcpf(s);
        if (q >= POST && q < POST + kFuseCh)
            pc[q - POST] = p;
    }
    const float coef = 2.f * alpha_over_n * beta;
#pragma unroll
    for (int t = 0; t < kFuseCh; ++t) {
        float cross = 0.f;
#pragma unroll
        for (int q = 0; q < SIZE; ++q)
            cross += r[t + q];
        gs[t][pos] = g[t + POST] * pc[t] - coef * a[t + POST + PRE] * cross;
        // (channels past C stage zeros or 0 offsets; phase 2 never reads them)
        if (mask_u8) {
            const uint32_t o = off(c0 + t);
            const int b = buf_ld_u8(rm, ((o & ~kOob) >> 2) | (o & kOob));
            const int du = b / kw;
            ms[t][pos] = b == 255 ? -1 : (wh0 + du) * W + ww0 + (b - du * kw);
        } else {
            ms[t][pos] = (int32_t)__builtin_bit_cast(uint32_t, buf_ld_f32(rm, off(c0 + t)));
        }
    }
}

// Phase 2 for one input position (h, w) and staged channel t: the sum, in
// row-major window order, of the pooled gradients of the covering windows
// whose winner it is.
template <int KS, int SS>
__device__ __forceinline__ float fuse_gather(const FuseBlock& f,
                                             const float (&gs)[kFuseCh][kFusePos],
                                             const int32_t (&ms)[kFuseCh][kFusePos], int t,
                                             int h, int w, int W, int OH, int OW, int kh, int kw,
                                             int sh, int sw, int ph, int pw)
{
    const int hw = h * W + w;
    const int i0 = max(0, (h + ph - kh + sh) / sh);
    const int i1 = min(OH - 1, (h + ph) / sh);
    const int j0 = max(0, (w + pw - kw + sw) / sw);
    const int j1 = min(OW - 1, (w + pw) / sw);
    float sum = 0.f;
    if constexpr (KS > 0) {
        // the covering windows (at most T x T), read first with their
        // indices clamped into the staged rows, then added in row-major
        // order where valid and routed here
        constexpr int T = (KS + SS - 1) / SS;
        int m[T][T];
        float g[T][T];
#pragma unroll
        for (int di = 0; di < T; ++di)
#pragma unroll
            for (int dj = 0; dj < T; ++dj) {
                const int o = (min(i0 + di, f.i_hi) - f.i_lo) * OW + min(j0 + dj, OW - 1);
                m[di][dj] = ms[t][o];
                g[di][dj] = gs[t][o];
            }
#pragma unroll
        for (int di = 0; di < T; ++di)
#pragma unroll
            for (int dj = 0; dj < T; ++dj)
                if (i0 + di <= i1 && j0 + dj <= j1 && m[di][dj] == hw)
                    sum += g[di][dj];
    } else {
        for (int ii = i0; ii <= i1; ++ii)
            for (int jj = j0; jj <= j1; ++jj) {
                const int o = (ii - f.i_lo) * OW + jj;
                if (ms[t][o] == hw)
                    sum += gs[t][o];
            }
    }
    return sum;
}

// Phase 2 for the 3x3 / stride-2 window, four input positions at a time:
// the positions (2a + dy - ph, 2b + dx - pw), dy, dx in {0, 1}, are covered
// only by windows among rows a - 1, a and columns b - 1, b (row a - 1 only
// for dy = 0, column b - 1 only for dx = 0), so the four records are read
// once for all four, and each position adds its routed gradients in the
// row-major window order of fuse_gather: the same sums, a quarter of the
// LDS reads and of the index arithmetic.
struct QuadMap {
    int a_lo, nar, b_lo, nbc, groups, grp, bc;
};

__device__ __forceinline__ QuadMap quad_map(const FuseBlock& f, int W, int ph, int pw)
{
    QuadMap q;
    q.a_lo = (f.y_lo + ph) >> 1;
    q.nar = ((f.y_hi + ph) >> 1) - q.a_lo + 1;
    q.b_lo = pw >> 1;
    q.nbc = ((W - 1 + pw) >> 1) - q.b_lo + 1;   // <= 129 for W <= 256
    q.groups = 256 / q.nbc;
    q.grp = threadIdx.x / q.nbc;
    q.bc = threadIdx.x - q.grp * q.nbc;
    return q;
}

__device__ __forceinline__ void fuse_gather_quad(const FuseBlock& f,
                                                 const float (&gs)[kFuseCh][kFusePos],
                                                 const int32_t (&ms)[kFuseCh][kFusePos],
                                                 int t, int a, int b, int W, int OH, int OW,
                                                 int ph, int pw, float (&out)[2][2])
{
    float g[2][2];
    int m[2][2];
    bool ok[2][2];
#pragma unroll
    for (int di = 0; di < 2; ++di)
#pragma unroll
        for (int dj = 0; dj < 2; ++dj) {
            const int i = a - 1 + di, j = b - 1 + dj;
            ok[di][dj] = i >= 0 && i < OH && j >= 0 && j < OW;
            // (clamped into the staged rows: a window a position outside
            // the strip would need is read but never used)
            const int o = (min(max(i, f.i_lo), f.i_hi) - f.i_lo) * OW + min(max(j, 0), OW - 1);
            g[di][dj] = gs[t][o];
            m[di][dj] = ms[t][o];
        }
#pragma unroll
    for (int dy = 0; dy < 2; ++dy)
#pragma unroll
        for (int dx = 0; dx < 2; ++dx) {
            const int hw = (2 * a + dy - ph) * W + 2 * b + dx - pw;
            float sum = 0.f;
#pragma unroll
            for (int di = dy; di < 2; ++di)
#pragma unroll
                for (int dj = dx; dj < 2; ++dj) {
                    if (ok[di][dj] && m[di][dj] == hw)
                        sum += g[di][dj];
                }
            out[dy][dx] = sum;
        }
}

template <int KS, int SS, int SIZE>
__global__ void __launch_bounds__(256)
lrn_pool_backward_kernel(const float* __restrict__ a_in, const float* __restrict__ g_in,
                         const int32_t* __restrict__ mask, float* __restrict__ dx, int N, int C, int H, int W, int OH, int OW,
                         int kh_, int kw_, int sh_, int sw_, int ph, int pw, int yrows,
                         int nstrips, int nchunks, float alpha_over_n, float beta, float k,
                         int mask_u8)
{
    __shared__ float gs[kFuseCh][kFusePos];
    __shared__ int32_t ms[kFuseCh][kFusePos];
    const int kh = KS ? KS : kh_, kw = KS ? KS : kw_;
    const int sh = SS ? SS : sh_, sw = SS ? SS : sw_;
    const FuseBlock f = fuse_block(H, OH, kh, sh, ph, yrows, nstrips, nchunks);
    fuse_stage_pooled_grad<SIZE>(f, a_in, g_in, mask, gs, ms, N, C, OH, OW, alpha_over_n, beta,
                                 k, mask_u8, W, kw, sh, sw, ph, pw);
    __syncthreads();
    if constexpr (KS == 3 && SS == 2) {
        // phase 2: thread -> one column pair b and every g-th row pair a
        const QuadMap qm = quad_map(f, W, ph, pw);
        if (qm.grp >= qm.groups)
            return;
        const int HW = H * W;
        for (int t = 0; t < kFuseCh; ++t) {
            const int ch = f.c0 + t;
            if (ch >= C)
                break;
            float* dplane = dx + ((size_t)f.n * C + ch) * HW;
            for (int ar = qm.grp; ar < qm.nar; ar += qm.groups) {
                const int a = qm.a_lo + ar, b = qm.b_lo + qm.bc;
                float q[2][2];
                fuse_gather_quad(f, gs, ms, t, a, b, W, OH, OW, ph, pw, q);
#pragma unroll
                for (int dy = 0; dy < 2; ++dy)
#pragma unroll
                    for (int ex = 0; ex < 2; ++ex) {
                        const int h = 2 * a + dy - ph, w = 2 * b + ex - pw;
                        if (h >= f.y_lo && h <= f.y_hi && w >= 0 && w < W)
                            dplane[h * W + w] = q[dy][ex];
                    }
            }
        }
        return;
    }
    // phase 2: thread -> one input column w (threads past the last full group
    // of W columns idle) and every g-th row of each channel
    const int groups = 256 / W;             // W <= 256 (the staged rows hold >= 1 row)
    const int grp = threadIdx.x / W;
    const int w = threadIdx.x - grp * W;
    if (grp >= groups)
        return;
    const int ny = f.y_hi - f.y_lo + 1;
    const int HW = H * W;
    for (int t = 0; t < kFuseCh; ++t) {
        const int ch = f.c0 + t;
        if (ch >= C)
            break;
        float* dplane = dx + ((size_t)f.n * C + ch) * HW;
        for (int hh = grp; hh < ny; hh += groups) {
            const int h = f.y_lo + hh;
            dplane[h * W + w] = fuse_gather<KS, SS>(f, gs, ms, t, h, w, W, OH, OW, kh, kw,
                                                          sh, sw, ph, pw);
        }
    }
}

// The same backward written straight into the bf16 top-gradient staging of
// the convolution below the pool (the layer whose output the pool read):
// Dh[n][h + tb][w + lb][g * Kgp + k] = bf16(D[n][g * Kg + k][h][w]) with
// D = the gathered gradient, times [relu_top > 0] when `relu_top` (the
// convolution's output) is given: the ReLU's backward, when the pool did not
// fold it.  A block's 16 channels lie in one
// group (Kg % 16 == 0), so each input position stores them as two 16-byte
// chunks.  The fp32 values are also summed per channel over the block's
// positions (each thread its own positions in row order, a fixed butterfly
// over each wave, then the four waves in order): sums[(g * Kg + k) * T +
// n * nstrips + strip], T = N * nstrips, the bias-gradient partials.  The staging grid's
// border is written by dh_zero_border_kernel.
template <int KS, int SS, int SIZE>
__global__ void __launch_bounds__(256)
lrn_pool_backward_bf16_kernel(const float* __restrict__ a_in, const float* __restrict__ g_in,
                              const int32_t* __restrict__ mask, const float* __restrict__ relu_top, uint16_t* __restrict__ Dh,
                              float* __restrict__ sums, int N, int C, int H, int W, int OH, int OW,
                              int kh_, int kw_, int sh_, int sw_, int ph, int pw, int yrows,
                              int nstrips, int nchunks, float alpha_over_n, float beta, float k,
                              int Kg, int Kgp, int Ktot, int DHp, int DWp, int tb, int lb,
                              int mask_u8)
{
    __shared__ float gs[kFuseCh][kFusePos];
    __shared__ int32_t ms[kFuseCh][kFusePos];
    const int kh = KS ? KS : kh_, kw = KS ? KS : kw_;
    const int sh = SS ? SS : sh_, sw = SS ? SS : sw_;
    const FuseBlock f = fuse_block(H, OH, kh, sh, ph, yrows, nstrips, nchunks);
    fuse_stage_pooled_grad<SIZE>(f, a_in, g_in, mask, gs, ms, N, C, OH, OW, alpha_over_n, beta,
                                 k, mask_u8, W, kw, sh, sw, ph, pw);
    __syncthreads();
    const int groups = 256 / W;
    const int grp = threadIdx.x / W;
    const int w = threadIdx.x - grp * W;
    const int ny = f.y_hi - f.y_lo + 1;
    const int HW = H * W;
    const int g = f.c0 / Kg;
    const int cp0 = g * Kgp + (f.c0 - g * Kg);
    const uint32_t tbytes = relu_top ? (uint32_t)(N * C * HW) * 4u : 0u;
    const __amdgpu_buffer_rsrc_t rt = make_rsrc(relu_top, tbytes);
    float bsum[kFuseCh];
#pragma unroll
    for (int t = 0; t < kFuseCh; ++t)
        bsum[t] = 0.f;
    if constexpr (KS == 3 && SS == 2) {
        // thread -> one column pair b and every g-th row pair a; each of
        // the four positions stores its 16 channels as two 16-byte chunks
        const QuadMap qm = quad_map(f, W, ph, pw);
        for (int ar = qm.grp; qm.grp < qm.groups && ar < qm.nar; ar += qm.groups) {
            const int a = qm.a_lo + ar, b = qm.b_lo + qm.bc;
            bool in[2][2];
#pragma unroll
            for (int dy = 0; dy < 2; ++dy)
#pragma unroll
                for (int ex = 0; ex < 2; ++ex) {
                    const int h = 2 * a + dy - ph, w = 2 * b + ex - pw;
                    in[dy][ex] = h >= f.y_lo && h <= f.y_hi && w >= 0 && w < W;
                }
            uint32_t packed[2][2][kFuseCh / 2];
#pragma unroll
            for (int t = 0; t < kFuseCh; t += 2) {
                float q[2][2][2];
                fuse_gather_quad(f, gs, ms, t, a, b, W, OH, OW, ph, pw, q[0]);
                fuse_gather_quad(f, gs, ms, t + 1, a, b, W, OH, OW, ph, pw, q[1]);
#pragma unroll
                for (int dy = 0; dy < 2; ++dy)
#pragma unroll
                    for (int ex = 0; ex < 2; ++ex) {
                        float v[2] = {q[0][dy][ex], q[1][dy][ex]};
                        if (relu_top) {
                            const int h = 2 * a + dy - ph, w = 2 * b + ex - pw;
#pragma unroll
                            for (int u = 0; u < 2; ++u) {
                                // (a NaN output masks too)
                                const uint32_t o =
                                    ((uint32_t)(((f.n * C + f.c0 + t + u) * H + h) * W + w) * 4u) |
                                    ((uint32_t)!in[dy][ex] << 31);
                                v[u] = buf_ld_f32(rt, o) > 0.f ? v[u] : 0.f;
                            }
                        }
                        if (in[dy][ex]) {
                            bsum[t] += v[0];
                            bsum[t + 1] += v[1];
                        }
                        packed[dy][ex][t / 2] = f32x2_to_bf16x2_rne(v[0], v[1]);
                    }
            }
#pragma unroll
            for (int dy = 0; dy < 2; ++dy)
#pragma unroll
                for (int ex = 0; ex < 2; ++ex) {
                    if (!in[dy][ex])
                        continue;
                    const int h = 2 * a + dy - ph, w = 2 * b + ex - pw;
                    u32x4* dst =
                        (u32x4*)&Dh[(((size_t)f.n * DHp + h + tb) * DWp + w + lb) * Ktot + cp0];
                    const uint32_t* pk = packed[dy][ex];
                    dst[0] = u32x4{pk[0], pk[1], pk[2], pk[3]};
                    dst[1] = u32x4{pk[4], pk[5], pk[6], pk[7]};
                }
        }
    } else if (grp < groups) {
        for (int hh = grp; hh < ny; hh += groups) {
            const int h = f.y_lo + hh;
            uint32_t packed[kFuseCh / 2];
#pragma unroll
            for (int t = 0; t < kFuseCh; t += 2) {
                float v[2];
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                    v[u] = fuse_gather<KS, SS>(f, gs, ms, t + u, h, w, W, OH, OW, kh, kw,
                                                     sh, sw, ph, pw);
                    if (relu_top) {
                        // (a NaN output masks too)
                        const uint32_t o = (uint32_t)(((f.n * C + f.c0 + t + u) * H + h) * W + w);
                        v[u] = buf_ld_f32(rt, o * 4u) > 0.f ? v[u] : 0.f;
                    }
                    bsum[t + u] += v[u];
                }
                packed[t / 2] = f32x2_to_bf16x2_rne(v[0], v[1]);
            }
            u32x4* dst = (u32x4*)&Dh[(((size_t)f.n * DHp + h + tb) * DWp + w + lb) * Ktot + cp0];
            dst[0] = u32x4{packed[0], packed[1], packed[2], packed[3]};
            dst[1] = u32x4{packed[4], packed[5], packed[6], packed[7]};
        }
    }
    // bias-gradient partials: per channel a wave butterfly (fixed), then the
    // four waves' sums added in wave order
    __shared__ float red[kFuseCh][4];
    const int wave = threadIdx.x >> 6;
#pragma unroll
    for (int t = 0; t < kFuseCh; ++t) {
        const float v = wave_sum(bsum[t]);
        if ((threadIdx.x & 63) == 0)
            red[t][wave] = v;
    }
    __syncthreads();
    const int t = threadIdx.x;
    if (t < kFuseCh && f.c0 + t < C) {
        const size_t T = (size_t)N * nstrips;
        sums[(size_t)(f.c0 + t) * T + (size_t)f.n * nstrips + f.strip] =
            ((red[t][0] + red[t][1]) + red[t][2]) + red[t][3];
    }
}

// Zeros of the bf16 top-gradient staging grid outside the image: the rows
// above and below it and the columns left and right of it, every channel, as
// 16-byte stores.  One thread per (image, border pixel, 8-channel chunk).
__global__ void __launch_bounds__(256)
dh_zero_border_kernel(uint16_t* __restrict__ Dh, int N, int DHp, int DWp, int tb, int lb, int H,
                      int W, int Ktot, long total)
{
    const long e = blockIdx.x * 256L + threadIdx.x;
    if (e >= total)
        return;
    const int chunks = Ktot / 8;
    const int border = DHp * DWp - H * W;
    const int c8 = (int)(e % chunks);
    const long pe = e / chunks;
    const int b = (int)(pe % border);
    const int n = (int)(pe / border);
    // border pixels in row-major order: tb full rows, then H rows of the
    // (DWp - W) side pixels, then the full rows below
    const int side = DWp - W;
    int hp, wp;
    if (b < tb * DWp) {
        hp = b / DWp;
        wp = b - hp * DWp;
    } else if (b < tb * DWp + H * side) {
        const int r = b - tb * DWp;
        hp = tb + r / side;
        const int j = r - (r / side) * side;
        wp = j < lb ? j : W + j;
    } else {
        const int r = b - tb * DWp - H * side;
        hp = tb + H + r / DWp;
        wp = r - (r / DWp) * DWp;
    }
    *(u32x4*)&Dh[(((size_t)n * DHp + hp) * DWp + wp) * Ktot + 8 * c8] = u32x4{0u, 0u, 0u, 0u};
}

hipError_t launch_dh_zero_border(uint16_t* Dh, int N, int DHp, int DWp, int tb, int lb, int H,
                                 int W, int Ktot, hipStream_t s)
{
    if (Ktot % 8 != 0 || tb < 0 || lb < 0 || DHp < tb + H || DWp < lb + W)
        return hipErrorInvalidValue;
    const long border = (long)N * (DHp * DWp - H * W) * (Ktot / 8);
    if (border > 0)
        hipLaunchKernelGGL(dh_zero_border_kernel, dim3((unsigned)((border + 255) / 256)), dim3(256),
                           0, s, Dh, N, DHp, DWp, tb, lb, H, W, Ktot, border);
    return hipGetLastError();
}

// The backward's strip: `yrows` input rows whose covering pooled rows (at
// most 256 positions) are staged; 0 when even one row does not fit.
static int fused_backward_yrows(int H, int OH, int OW, int kh, int sh, int ph)
{
    for (int yr = H; yr >= 1; --yr) {
        // worst strip: pooled rows reached by yr consecutive input rows
        const int span = (yr - 1 + kh - 1) / sh + 1 + 1;
        if (min(span, OH) * OW <= kFusePos)
            return yr;
    }
    (void)ph;
    return 0;
}

bool pool_lrn_fusable(int H, int W, int OH, int OW, int kh, int sh, int ph, int size)
{
    // (the backward gives each thread one input column of a row group)
    return (size == 3 || size == 5) && W <= kFusePos &&
           fused_backward_yrows(H, OH, OW, kh, sh, ph) > 0;
}

hipError_t launch_lrn_pool_backward(const float* pooled, const float* top, const float* top_diff,
                                    const int32_t* mask, float* dx, int N, int C, int H, int W,
                                    int OH, int OW, int kh, int kw, int sh, int sw, int ph, int pw,
                                    int size, float alpha, float beta, float k, hipStream_t s,
                                    int mask_u8)
{
    if ((long)N * C * H * W == 0)
        return hipSuccess;
    const int yrows = fused_backward_yrows(H, OH, OW, kh, sh, ph);
    if (yrows == 0 || (size != 3 && size != 5) || (mask_u8 && kh * kw > 255))
        return hipErrorInvalidValue;
    const int nstrips = (H + yrows - 1) / yrows;
    const int nchunks = (C + kFuseCh - 1) / kFuseCh;
    const dim3 g((unsigned)((long)N * nchunks * nstrips));
    const float an = alpha / size;
#define FUSED_BWD(KS_, SS_, SZ_)                                                                  \
    hipLaunchKernelGGL((lrn_pool_backward_kernel<KS_, SS_, SZ_>), g, dim3(256), 0, s, pooled,    \
                       top_diff, mask, dx, N, C, H, W, OH, OW, kh, kw, sh, sw, ph, pw, yrows,   \
                       nstrips, nchunks, an, beta, k, mask_u8)
    const bool k32 = kh == 3 && kw == 3 && sh == 2 && sw == 2;
    if (size == 5) {
        if (k32)
            FUSED_BWD(3, 2, 5);
        else
            FUSED_BWD(0, 0, 5);
    } else {
        if (k32)
            FUSED_BWD(3, 2, 3);
        else
            FUSED_BWD(0, 0, 3);
    }
#undef FUSED_BWD
    return hipGetLastError();
}

int lrn_pool_backward_strips(int H, int OH, int OW, int kh, int sh, int ph)
{
    const int yrows = fused_backward_yrows(H, OH, OW, kh, sh, ph);
    return yrows > 0 ? (H + yrows - 1) / yrows : 0;
}

hipError_t launch_lrn_pool_backward_bf16(const float* pooled, const float* top,
                                         const float* top_diff, const int32_t* mask,
                                         const float* relu_top, uint16_t* Dh, float* sums, int N,
                                         int C, int H, int W, int OH, int OW, int kh, int kw,
                                         int sh, int sw, int ph, int pw, int size, float alpha,
                                         float beta, float k, int Kg, int Kgp, int Ktot, int DHp,
                                         int DWp, int tb, int lb, hipStream_t s, int mask_u8)
{
    if ((long)N * C * H * W == 0)
        return hipSuccess;
    const int yrows = fused_backward_yrows(H, OH, OW, kh, sh, ph);
    if (yrows == 0 || (size != 3 && size != 5) || Kg % kFuseCh != 0 || Ktot % 8 != 0 ||
        tb < 0 || lb < 0 || DHp < tb + H || DWp < lb + W || (mask_u8 && kh * kw > 255))
        return hipErrorInvalidValue;
    const hipError_t e = launch_dh_zero_border(Dh, N, DHp, DWp, tb, lb, H, W, Ktot, s);
    if (e != hipSuccess)
        return e;
    const int nstrips = (H + yrows - 1) / yrows;
    const int nchunks = C / kFuseCh;
    const dim3 g((unsigned)((long)N * nchunks * nstrips));
    const float an = alpha / size;
#define FUSED_BWD16(KS_, SS_, SZ_)                                                                \
    hipLaunchKernelGGL((lrn_pool_backward_bf16_kernel<KS_, SS_, SZ_>), g, dim3(256), 0, s,       \
                       pooled, top_diff, mask, relu_top, Dh, sums, N, C, H, W, OH, OW, kh, kw,   \
                       sh, sw, ph, pw, yrows, nstrips, nchunks, an, beta, k, Kg, Kgp, Ktot, DHp, \
                       DWp, tb, lb, mask_u8)
    const bool k32 = kh == 3 && kw == 3 && sh == 2 && sw == 2;
    if (size == 5) {
        if (k32)
            FUSED_BWD16(3, 2, 5);
        else
            FUSED_BWD16(0, 0, 5);
    } else {
        if (k32)
            FUSED_BWD16(3, 2, 3);
        else
            FUSED_BWD16(0, 0, 3);
    }
#undef FUSED_BWD16
    return hipGetLastError();
}

// --------------------------------------------------------------------- cast
// Eight values per thread and step: two 16-byte loads, one 16-byte store
// (both tensors are 16-byte aligned); the last count % 8 values one by one.
__global__ void __launch_bounds__(256)
cast_f32_bf16_kernel(const float* __restrict__ x, uint16_t* __restrict__ y, int64_t count)
{
    const int64_t n8 = count / 8;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t t0 = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    for (int64_t i = t0; i < n8; i += stride) {
        const float4 a = ((const float4*)x)[2 * i];
        const float4 b = ((const float4*)x)[2 * i + 1];
        u32x4 o;
        o[0] = f32x2_to_bf16x2_rne(a.x, a.y);
        o[1] = f32x2_to_bf16x2_rne(a.z, a.w);
        o[2] = f32x2_to_bf16x2_rne(b.x, b.y);
        o[3] = f32x2_to_bf16x2_rne(b.z, b.w);
        ((u32x4*)y)[i] = o;
    }
    for (int64_t e = 8 * n8 + t0; e < count; e += stride)
        y[e] = f32_to_bf16_rne(x[e]);
}

hipError_t launch_cast_f32_bf16(const float* x, uint16_t* y, int64_t count, hipStream_t s)
{
    if (count == 0)
        return hipSuccess;
    hipLaunchKernelGGL(cast_f32_bf16_kernel, dim3(grid_for(std::max<int64_t>(count / 8, 1))),
                       dim3(256), 0, s, x, y, count);
    return hipGetLastError();
}

}  // namespace caffe_hip
