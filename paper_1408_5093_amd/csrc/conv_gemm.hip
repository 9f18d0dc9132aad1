// conv_gemm.hip -- implicit-GEMM convolution on gfx950 fp32 MFMA.
//
// Forward pass and data gradient of the convolution layer (the paper's layer
// definition, Sec. 3.2).  The lowering of the input to a dense contraction
// ("im2col") is never materialised: each workgroup gathers its slice of the
// lowered matrix straight from the NCHW blob into LDS, then runs the
// contraction on the matrix cores.
//
// GEMM per group g:  C[m][col] = sum_r A[g][m][r] * B_g[r][col]
//   r   = (c, u, v)  over Cin_g x kh x kw      (reduction, staged TK at a time)
//   col = (n, i, j)  over N x OH x OW          (columns, TN per workgroup)
//   B_g[r][col] = X[n][g*Cin_g + c][i*sh - ph + u][j*sw - pw + v]   (0 outside)
//
// Pipeline per workgroup: the global loads of stage s+1 are issued into
// registers before the MFMAs of stage s run out of LDS buffer s%2, then the
// registers go to LDS buffer (s+1)%2; one barrier per stage.
//
// MFMA operand layouts (single-block f32 variants):
//   32x32x2 : A lane l -> (row l%32, k l/32), B lane l -> (k l/32, col l%32),
//             D reg q -> (row 8*(q/4) + 4*(l/32) + q%4, col l%32)
//   16x16x4 : A lane l -> (row l%16, k l/16), B lane l -> (k l/16, col l%16),
//             D reg q -> (row 4*(l/16) + q, col l%16)
#include "device_common.h"
#include "kernels.h"

namespace caffe_hip {

template <int MT>
struct Mfma;

template <>
struct Mfma<32> {
    static constexpr int kStep = 2;
    static constexpr int kRegs = 16;
    typedef floatx16 acc_t;
    static __device__ __forceinline__ acc_t run(float a, float b, acc_t c)
    {
        return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
    }
    static __device__ __forceinline__ int row(int q, int lane)
    {
        return 8 * (q >> 2) + 4 * (lane >> 5) + (q & 3);
    }
};

template <>
struct Mfma<16> {
    static constexpr int kStep = 4;
    static constexpr int kRegs = 4;
    typedef floatx4 acc_t;
    static __device__ __forceinline__ acc_t run(float a, float b, acc_t c)
    {
        return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
    }
    static __device__ __forceinline__ int row(int q, int lane) { return 4 * (lane >> 4) + q; }
};

template <int MT, int WM, int WN, int MI, int NI, int TK, int KH, int KW, int SH, int SW, int EPI,
          bool TAP, bool MASK>
__global__ void __launch_bounds__(64 * WM * WN)
conv_gemm_f32_kernel(const ConvGemmParams p)
{
    typedef Mfma<MT> Op;
    constexpr int NT = 64 * WM * WN;
    constexpr int TM = WM * MI * MT;
    constexpr int TN = WN * NI * MT;
    constexpr int EA = TM * TK / NT;  // A elements per thread per stage
    constexpr int EB = TN * TK / NT;  // B elements per thread per stage
    constexpr int KS = TK / Op::kStep;
    static_assert(TM * TK % NT == 0 && TN * TK % NT == 0, "tile/thread mismatch");
    static_assert(NT % TK == 0, "A mapping needs TK | NT");
    static_assert(TN % 64 == 0 && (NT % TN == 0 || TN % NT == 0), "B mapping");
    static_assert(TK % Op::kStep == 0, "stage depth");
    constexpr int BC = TN > NT ? TN / NT : 1;  // distinct B columns per thread
    // Row strides: A rows are written with lanes along k, so a stride of
    // 2 (mod 32) keeps those writes conflict-free.  The 16x16x4 fragments read
    // four k rows at once, so B rows then get a stride of 16 (mod 32).
    constexpr int PADA = 2;
    constexpr int PADB = MT == 16 ? 16 : 0;

    __shared__ float As[2][TK][TM + PADA];
    __shared__ float Bs[2][TK][TN + PADB];

    const int kh = KH ? KH : p.kh;
    const int kw = KW ? KW : p.kw;
    const int sh = SH ? SH : p.sh;
    const int sw = SW ? SW : p.sw;
    const int khw = kh * kw;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave % WM;
    const int wn = wave / WM;
    // XCD-contiguous tile order: the hardware deals workgroups to the 8 XCDs
    // round-robin, so workgroup L runs on XCD L % 8; tile T = (L % 8) * per_xcd
    // + L / 8 gives each XCD a contiguous run of tiles.  Row tiles vary
    // fastest, so the tiles that share a column block of the gathered operand
    // run together on one XCD and share its L2.
    const int n_mt = (p.M + TM - 1) / TM;
    const int n_ct = (p.Ncol + TN - 1) / TN;
    const int per_xcd = gridDim.x >> 3;
    const int T = p.xcd_order ? (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3) : blockIdx.x;
    if (T >= n_mt * n_ct * p.G)
        return;
    const int mt = T % n_mt;
    const int ct = (T / n_mt) % n_ct;
    const int g = T / (n_mt * n_ct);
    const int m0 = mt * TM;
    const int n0 = ct * TN;
    const int M = p.M, R = p.R;
    const int IH = p.IH, IW = p.IW, IHW = IH * IW;
    const int OHW = p.OH * p.OW;
    const int Cin_g = p.Cin_g;

    const __amdgpu_buffer_rsrc_t ra = make_rsrc(p.A, p.A_bytes);
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(p.X, p.X_bytes);

    // ---- A mapping: k = tid % TK, m = tid / TK + (NT / TK) * q
    const int a_k = tid % TK;
    const int a_m = tid / TK;
    // A rows m0 + a_m + (NT/TK)*q, byte offsets linear in q.  Rows past M need
    // no mask: they only feed accumulator rows the epilogue never stores, and
    // their loads stay inside the weights or read 0.
    const uint32_t a_base4 = (uint32_t)((g * M + m0 + a_m) * R) * 4u;

    // ---- B mapping: column(s) fixed per thread, reduction rows vary
    int b_base[BC], b_ih0[BC], b_iw0[BC];
#pragma unroll
    for (int cc = 0; cc < BC; ++cc) {
        const int col = n0 + (TN > NT ? tid + NT * cc : tid % TN);
        if (col < p.Ncol) {
            const int n = col / OHW;
            const int pix = col - n * OHW;
            const int i = pix / p.OW;
            const int j = pix - i * p.OW;
            b_ih0[cc] = i * sh - p.ph;
            b_iw0[cc] = j * sw - p.pw;
            b_base[cc] = (n * p.Cin + g * Cin_g) * IHW + b_ih0[cc] * IW + b_iw0[cc];
        } else {
            b_ih0[cc] = -(1 << 28);  // fails every bounds check
            b_iw0[cc] = 0;
            b_base[cc] = 0;
        }
    }
    auto b_row = [&](int q) { return TN > NT ? q / BC : tid / TN + (NT / TN) * q; };
    auto b_cc = [&](int q) { return TN > NT ? q % BC : 0; };

    float rA[EA], rB[EB];

    auto load_a = [&](int kbase) {
        const int r = kbase + a_k;
        // the channel-blocked order covers R in whole stages (R % TK == 0)
        const uint32_t rbad = TAP ? 0u : (uint32_t)(r >= R) << 31;
        const uint32_t r4 = a_base4 + (uint32_t)r * 4u;
#pragma unroll
        for (int q = 0; q < EA; ++q)
            rA[q] = buf_ld_f32(ra, (r4 + (uint32_t)((NT / TK) * q * R) * 4u) | rbad);
    };

    // Channel-blocked reduction order r = (c / TK, u, v, c % TK): Cin_g is a
    // multiple of TK, so a stage covers TK channels of a single tap (u, v);
    // the tap's bounds check and address are computed once per column per
    // stage.  All taps of a channel block run back to back, so a workgroup
    // re-reads the same TK channel planes (from L1/L2) tap after tap.
    auto load_b_tap = [&](int u, int v, int c0) {
        uint32_t voff[BC];
#pragma unroll
        for (int cc = 0; cc < BC; ++cc) {
            const int ih = b_ih0[cc] + u;
            const int iw = b_iw0[cc] + v;
            const bool ok = (unsigned)ih < (unsigned)IH && (unsigned)iw < (unsigned)IW;
            voff[cc] = ok ? (uint32_t)(b_base[cc] + u * IW + v) * 4u : kOob;
        }
#pragma unroll
        for (int q = 0; q < EB; ++q) {
            const uint32_t coff = (uint32_t)((c0 + b_row(q)) * IHW) * 4u;
            rB[q] = buf_ld_f32(rx, voff[b_cc(q)] + coff);
        }
    };

    // Channel-major order r = (c, u, v) for any Cin_g.  The tap decomposition
    // is wave-uniform (scalar).  Out-of-range taps get an offset with bit 31
    // set; a wave whose columns all have their whole window inside the image
    // (every wave of an unpadded layer) skips the per-tap bounds test.
    bool b_inside = true;
#pragma unroll
    for (int cc = 0; cc < BC; ++cc)
        b_inside = b_inside && b_ih0[cc] >= 0 && b_ih0[cc] + kh <= IH && b_iw0[cc] >= 0 &&
                   b_iw0[cc] + kw <= IW;
    const bool b_all_inside = __all(b_inside);
    auto load_b_any = [&](int kbase) {
        if (b_all_inside) {
#pragma unroll
            for (int q = 0; q < EB; ++q) {
                const int r = __builtin_amdgcn_readfirstlane(kbase + b_row(q));
                const int c = r / khw;
                const int rr = r - c * khw;
                const int u = rr / kw;
                const int v = rr - u * kw;
                const uint32_t rbad = r < R ? 0u : kOob;
                rB[q] = buf_ld_f32(rx, ((uint32_t)(b_base[b_cc(q)] + c * IHW + u * IW + v) * 4u) |
                                           rbad);
            }
        } else {
#pragma unroll
            for (int q = 0; q < EB; ++q) {
                const int cc = b_cc(q);
                const int r = __builtin_amdgcn_readfirstlane(kbase + b_row(q));
                const int c = r / khw;
                const int rr = r - c * khw;
                const int u = rr / kw;
                const int v = rr - u * kw;
                const int ih = b_ih0[cc] + u;
                const int iw = b_iw0[cc] + v;
                const uint32_t bad = ((uint32_t)(r >= R) | (uint32_t)((unsigned)ih >= (unsigned)IH) |
                                      (uint32_t)((unsigned)iw >= (unsigned)IW)) << 31;
                rB[q] = buf_ld_f32(rx, ((uint32_t)(b_base[cc] + c * IHW + u * IW + v) * 4u) | bad);
            }
        }
    };

    auto store_stage = [&](int buf) {
#pragma unroll
        for (int q = 0; q < EA; ++q)
            As[buf][a_k][a_m + (NT / TK) * q] = rA[q];
#pragma unroll
        for (int q = 0; q < EB; ++q) {
            const int col = TN > NT ? tid + NT * b_cc(q) : tid % TN;
            Bs[buf][b_row(q)][col] = rB[q];
        }
    };

    // The forward pass starts every accumulator at its row's bias (the sum
    // then runs bias + products, as in the layer's definition); a null bias
    // is a zero-record buffer that reads 0.
    typename Op::acc_t acc[MI][NI];
#pragma unroll
    for (int mi = 0; mi < MI; ++mi) {
        typename Op::acc_t init{};
        if constexpr (EPI == 0) {
            const __amdgpu_buffer_rsrc_t rbias =
                make_rsrc(p.bias, p.bias ? (uint32_t)(p.G * M) * 4u : 0u);
#pragma unroll
            for (int q = 0; q < Op::kRegs; ++q) {
                const int m = m0 + wm * MI * MT + mi * MT + Op::row(q, lane);
                init[q] = buf_ld_f32(rbias, m < M ? (uint32_t)(g * M + m) * 4u : kOob);
            }
        }
#pragma unroll
        for (int ni = 0; ni < NI; ++ni)
            acc[mi][ni] = init;
    }

    const int nst = (R + TK - 1) / TK;
    // blocked walk state: stage s covers tap (tu, tv) of channels tc .. tc + TK - 1.
    // It is updated in the loop body itself: captured by reference in a
    // lambda, it was kept in scratch memory, and the scratch accesses' waits
    // also stalled on the next stage's global loads.
    int tu = 0, tv = 0, tc = 0;

    load_a(0);
    if constexpr (TAP)
        load_b_tap(0, 0, 0);
    else
        load_b_any(0);
    store_stage(0);
    __syncthreads();

    const int arow = wm * MI * MT + lane % MT;
    const int bcol = wn * NI * MT + lane % MT;
    const int kl = lane / MT;

    for (int s = 0; s < nst; ++s) {
        const int cur = s & 1;
        if (s + 1 < nst) {
            load_a((s + 1) * TK);
            if constexpr (TAP) {
                if (p.blocked) {  // (c / TK, u, v, c % TK)
                    if (++tv == kw) {
                        tv = 0;
                        if (++tu == kh) {
                            tu = 0;
                            tc += TK;
                        }
                    }
                } else {          // (u, v, c)
                    tc += TK;
                    if (tc == Cin_g) {
                        tc = 0;
                        if (++tv == kw) {
                            tv = 0;
                            ++tu;
                        }
                    }
                }
                load_b_tap(tu, tv, tc);
            } else {
                load_b_any((s + 1) * TK);
            }
        }
        // Rolling fragment prefetch: the LDS reads of k-step ks + PF are issued
        // before the MFMAs of k-step ks (a ring of PF + 1 fragment sets).  The
        // scheduling barriers pin that order; left alone, the scheduler trades
        // it for fewer registers and waits on LDS before every k-step.
        constexpr int PF = KS > 2 ? 2 : KS - 1;
        float fa[PF + 1][MI], fb[PF + 1][NI];
        auto read_frag = [&](int ks, int slot) {
#pragma unroll
            for (int mi = 0; mi < MI; ++mi)
                fa[slot][mi] = As[cur][ks * Op::kStep + kl][arow + mi * MT];
#pragma unroll
            for (int ni = 0; ni < NI; ++ni)
                fb[slot][ni] = Bs[cur][ks * Op::kStep + kl][bcol + ni * MT];
        };
#pragma unroll
        for (int ks = 0; ks < PF; ++ks)
            read_frag(ks, ks);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            if (ks + PF < KS)
                read_frag(ks + PF, (ks + PF) % (PF + 1));
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int mi = 0; mi < MI; ++mi)
#pragma unroll
                for (int ni = 0; ni < NI; ++ni)
                    acc[mi][ni] = Op::run(fa[ks % (PF + 1)][mi], fb[ks % (PF + 1)][ni],
                                          acc[mi][ni]);
            __builtin_amdgcn_sched_barrier(0);
        }
        if (s + 1 < nst)
            store_stage(cur ^ 1);
        __syncthreads();
    }

    // ---- epilogue (branch-free: masked lanes store to an out-of-range offset)
    const __amdgpu_buffer_rsrc_t ry = make_rsrc(p.Y, p.Y_bytes);
    // Masks are folded into the offsets with integer ops (bit 31 = past the
    // buffer, dropped by the hardware): short-circuit tests here become
    // divergent branches and make the compiler copy every accumulator out of
    // the AGPRs at once.
    if constexpr (EPI == 0) {
        int cbase[NI];
        uint32_t cbad[NI];
#pragma unroll
        for (int ni = 0; ni < NI; ++ni) {
            const int col = n0 + bcol + ni * MT;
            const int n = col / OHW;
            const int pix = col - n * OHW;
            cbase[ni] = n * p.Cout * OHW + pix;
            cbad[ni] = (uint32_t)(col >= p.Ncol) << 31;
        }
#pragma unroll
        for (int mi = 0; mi < MI; ++mi) {
#pragma unroll
            for (int ni = 0; ni < NI; ++ni) {
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int q = 0; q < Op::kRegs; ++q) {
                    const int m = m0 + wm * MI * MT + mi * MT + Op::row(q, lane);
                    const int oc = g * M + m;
                    const float z = acc[mi][ni][q];
                    // ReLU: non-positive values (NaN included) become 0; without
                    // ReLU every value passes unchanged
                    const float v = z > 0.f ? z : (p.relu ? 0.f : z);
                    const uint32_t off = ((uint32_t)(cbase[ni] + oc * OHW) * 4u) | cbad[ni] |
                                         ((uint32_t)(m >= M) << 31);
                    buf_st_f32(v, ry, off);
                }
            }
        }
    } else {
        const int pss = p.psh * p.psw;
        const int OutHW = p.OutH * p.OutW;
        const __amdgpu_buffer_rsrc_t rom = make_rsrc(MASK ? p.Omask : p.Y, p.Y_bytes);
        int cb[NI], hb[NI], wb[NI];
#pragma unroll
        for (int ni = 0; ni < NI; ++ni) {
            const int col = n0 + bcol + ni * MT;
            const bool cok = col < p.Ncol;
            const int n = cok ? col / OHW : 0;
            const int pix = col - n * OHW;
            const int a = pix / p.OW;
            const int b = pix - a * p.OW;
            hb[ni] = cok ? p.psh * (a + p.a0h) - p.oph : -(1 << 28);
            wb[ni] = p.psw * (b + p.a0w) - p.opw;
            cb[ni] = (n * p.Cout + g * p.Cg_out) * OutHW;
        }
#pragma unroll
        for (int mi = 0; mi < MI; ++mi) {
#pragma unroll
            for (int q = 0; q < Op::kRegs; ++q) {
                const int m = m0 + wm * MI * MT + mi * MT + Op::row(q, lane);
                int c = m, fh = 0, fw = 0;
                if (pss != 1) {
                    c = m / pss;
                    const int fr = m - c * pss;
                    fh = fr / p.psw;
                    fw = fr - fh * p.psw;
                }
#pragma unroll
                for (int ni = 0; ni < NI; ++ni) {
                    const int h = hb[ni] + fh;
                    const int w = wb[ni] + fw;
                    const uint32_t bad = ((uint32_t)(m >= M) |
                                          (uint32_t)((unsigned)h >= (unsigned)p.OutH) |
                                          (uint32_t)((unsigned)w >= (unsigned)p.OutW))
                                         << 31;
                    const uint32_t off =
                        ((uint32_t)(cb[ni] + c * OutHW + h * p.OutW + w) * 4u) | bad;
                    float v = acc[mi][ni][q];
                    if constexpr (MASK) {
                        // backward of the ReLU that produced the gather target:
                        // keep the gradient only where that output was > 0
                        const float y = buf_ld_f32(rom, off);
                        v = y > 0.f ? v : 0.f;
                    }
                    buf_st_f32(v, ry, off);
                }
            }
        }
    }
}

// Forward weights in the channel-blocked order:
// Wp[o][((c / tk) * khw + t) * tk + c % tk] = W[o][c][t], t = u*kw + v.
__global__ void __launch_bounds__(256)
pack_weights_blocked_kernel(const float* __restrict__ W, float* __restrict__ Wp, int K, int Cg,
                            int khw, int tk, int blocked)
{
    const int total = K * Cg * khw;
    const int e = blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= total)
        return;
    const int R = Cg * khw;
    const int o = e / R;
    const int r = e - o * R;
    int c, t;
    if (blocked) {
        const int ci = r % tk;
        t = (r / tk) % khw;
        c = (r / (tk * khw)) * tk + ci;
    } else {
        t = r / Cg;
        c = r - t * Cg;
    }
    Wp[e] = W[(o * Cg + c) * khw + t];
}

hipError_t launch_pack_weights_blocked(const float* W, float* Wp, int K, int Cg, int khw, int tk,
                                       int blocked, hipStream_t s)
{
    const int total = K * Cg * khw;
    if (total == 0)
        return hipSuccess;
    hipLaunchKernelGGL(pack_weights_blocked_kernel, dim3((total + 255) / 256), dim3(256), 0, s, W,
                       Wp, K, Cg, khw, tk, blocked);
    return hipGetLastError();
}

// ------------------------------------------------------------------ launch
namespace {

struct TileShape {
    int mt, wm, wn, mi, ni, tk;
};
constexpr TileShape kTiles[TILE_COUNT] = {
    {32, 2, 2, 2, 2, 16},  // 128 x 128
    {32, 1, 4, 3, 2, 16},  // 96 x 256
    {16, 1, 4, 3, 4, 16},  // 48 x 256
    {32, 1, 4, 2, 2, 16},  // 64 x 256
    {32, 2, 2, 2, 2, 32},  // 128 x 128, 32-deep stages
};

template <int MT, int WM, int WN, int MI, int NI, int TK, int KH, int KW, int SH, int SW, int EPI,
          bool TAP, bool MASK>
hipError_t launch_one(const ConvGemmParams& p, hipStream_t s)
{
    constexpr int TM = WM * MI * MT, TN = WN * NI * MT;
    const int64_t tiles =
        (int64_t)((p.Ncol + TN - 1) / TN) * ((p.M + TM - 1) / TM) * p.G;
    const int64_t per_xcd = (tiles + 7) / 8;  // 8 XCDs; see the kernel's tile order
    hipLaunchKernelGGL(
        (conv_gemm_f32_kernel<MT, WM, WN, MI, NI, TK, KH, KW, SH, SW, EPI, TAP, MASK>),
        dim3((unsigned)(per_xcd * 8)), dim3(64 * WM * WN), 0, s, p);
    return hipGetLastError();
}

template <int MT, int WM, int WN, int MI, int NI, int TK, int EPI, bool MASK>
hipError_t launch_geom(const ConvGemmParams& p, bool tap, hipStream_t s)
{
    if (tap) {
        if (p.sh == 1 && p.sw == 1) {
            if (p.kh == 3 && p.kw == 3)
                return launch_one<MT, WM, WN, MI, NI, TK, 3, 3, 1, 1, EPI, true, MASK>(p, s);
            if (p.kh == 5 && p.kw == 5)
                return launch_one<MT, WM, WN, MI, NI, TK, 5, 5, 1, 1, EPI, true, MASK>(p, s);
        }
        return launch_one<MT, WM, WN, MI, NI, TK, 0, 0, 0, 0, EPI, true, MASK>(p, s);
    }
    if (EPI == 0 && p.kh == 11 && p.kw == 11 && p.sh == 4 && p.sw == 4)
        return launch_one<MT, WM, WN, MI, NI, TK, 11, 11, 4, 4, EPI, false, MASK>(p, s);
    return launch_one<MT, WM, WN, MI, NI, TK, 0, 0, 0, 0, EPI, false, MASK>(p, s);
}

template <int EPI, bool MASK>
hipError_t launch_tile(const ConvGemmParams& p, int tile, bool tap, hipStream_t s)
{
    switch (tile) {
    case TILE_128x128:
        return launch_geom<32, 2, 2, 2, 2, 16, EPI, MASK>(p, tap, s);
    case TILE_96x256:
        return launch_geom<32, 1, 4, 3, 2, 16, EPI, MASK>(p, tap, s);
    case TILE_48x256:
        return launch_geom<16, 1, 4, 3, 4, 16, EPI, MASK>(p, tap, s);
    case TILE_64x256:
        return launch_geom<32, 1, 4, 2, 2, 16, EPI, MASK>(p, tap, s);
    case TILE_128x128_K32:
        return launch_geom<32, 2, 2, 2, 2, 32, EPI, MASK>(p, tap, s);
    default:
        return hipErrorInvalidValue;
    }
}

}  // namespace

int gemm_tile_m(int tile)
{
    const TileShape& t = kTiles[tile];
    return t.wm * t.mi * t.mt;
}

int gemm_tile_n(int tile)
{
    const TileShape& t = kTiles[tile];
    return t.wn * t.ni * t.mt;
}

int gemm_tile_k(int tile) { return kTiles[tile].tk; }

hipError_t launch_conv_gemm_f32(const ConvGemmParams& p, int epi, int tile, bool tap_major,
                                hipStream_t s)
{
    if (p.Ncol == 0)
        return hipSuccess;
    if (tile < 0 || tile >= TILE_COUNT || (tap_major && p.Cin_g % kTiles[tile].tk != 0))
        return hipErrorInvalidValue;
    if (epi == 0)
        return launch_tile<0, false>(p, tile, tap_major, s);
    return p.Omask ? launch_tile<1, true>(p, tile, tap_major, s)
                   : launch_tile<1, false>(p, tile, tap_major, s);
}

}  // namespace caffe_hip
