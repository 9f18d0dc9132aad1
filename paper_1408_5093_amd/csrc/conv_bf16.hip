// conv_bf16.hip -- the convolution layer on bfloat16 operands with fp32
// accumulation and fp32 results: forward pass, data gradient and weight
// gradient (the roles of the paper's Sec. 3.2 layer definition) as implicit
// GEMMs on the gfx950 bf16 matrix instructions.
//
// The bf16 instructions take eight consecutive reduction elements per lane
//   v_mfma_f32_32x32x16_bf16: A lane l -> row l%32, k 8*(l/32) .. +7
//                             B lane l -> col l%32, k 8*(l/32) .. +7
//   v_mfma_f32_16x16x32_bf16: A lane l -> row l%16, k 8*(l/16) .. +7 (B alike)
// (the result layout is that of the fp32 variants), so every operand is
// staged in LDS with its reduction index contiguous, and fragments are read
// 16 bytes at a time.
//
// Operand staging.  The gathered operands are first rewritten in the caller's
// workspace as channel-contiguous ("NHWC") bf16 blobs, each group's channels
// padded with zeros to Cgp, a multiple of 8:
//   Xh[n][h][w][g*Cgp + c] = bottom[n][g*Cg + c][h][w]             (c < Cg, else 0)
//   Dh[n][i][j][g*Kgp + k] = bf16(top_diff [top > 0])[n][g*Kg + k][i][j]
// so that one 16-byte load brings 8 reduction elements (8 channels of one
// pixel).  The reductions then run tap-major, r = (u, v, c) with c fastest.
//   forward:        C[m][(n,i,j)] = sum_r Wp[g][m][r] * Xh[n][i*sh-ph+u][j*sw-pw+v][g*Cgp+c]
//   data gradient:  the phase-stacked GEMM of the fp32 path, gathering Dh
//   weight grad.:   P[m][(u,v,c)] = sum_(n,i,j) Dh[n][i][j][g*Kgp+m] * Xh[n][i*sh-ph+u][j*sw-pw+v][g*Cgp+c]
#include "device_common.h"
#include "kernels.h"

namespace caffe_hip {

typedef uint16_t bf16_t;

__device__ __forceinline__ u32x4 buf_ld_b128(__amdgpu_buffer_rsrc_t r, uint32_t byte_off)
{
    return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, 0));
}

__device__ __forceinline__ bf16x8 lds_frag(const bf16_t* p)
{
    return __builtin_bit_cast(bf16x8, *(const u32x4*)p);
}

template <int MT>
struct MfmaBf16;

template <>
struct MfmaBf16<32> {
    static constexpr int kK = 16;  // reduction depth of one instruction
    static constexpr int kRegs = 16;
    typedef floatx16 acc_t;
    static __device__ __forceinline__ acc_t run(bf16x8 a, bf16x8 b, acc_t c)
    {
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
    }
    static __device__ __forceinline__ int row(int q, int lane)
    {
        return 8 * (q >> 2) + 4 * (lane >> 5) + (q & 3);
    }
};

template <>
struct MfmaBf16<16> {
    static constexpr int kK = 32;
    static constexpr int kRegs = 4;
    typedef floatx4 acc_t;
    static __device__ __forceinline__ acc_t run(bf16x8 a, bf16x8 b, acc_t c)
    {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
    static __device__ __forceinline__ int row(int q, int lane) { return 4 * (lane >> 4) + q; }
};

// ------------------------------------------------------------ forward / dgrad
template <int MT, int WM, int WN, int MI, int NI, int TK, int EPI, bool MASK>
__global__ void __launch_bounds__(64 * WM * WN)
conv_gemm_bf16_kernel(const GemmBf16Params p)
{
    typedef MfmaBf16<MT> Op;
    constexpr int NT = 64 * WM * WN;
    constexpr int TM = WM * MI * MT;
    constexpr int TN = WN * NI * MT;
    constexpr int TB = TK / 8;       // 16-byte chunks of a row per stage
    constexpr int LD = TK + 8;       // LDS row length: 16 bytes of padding
    constexpr int CA = TM * TB;      // A chunks per stage
    constexpr int EA = (CA + NT - 1) / NT;
    static_assert(TN <= NT && NT % TN == 0, "B mapping: a thread owns one column");
    constexpr int BS = NT / TN;      // B chunk slots covered by one pass of the block
    static_assert(TB % BS == 0, "B mapping");
    constexpr int EB = TB / BS;      // B chunks per thread per stage
    constexpr int KS = TK / Op::kK;
    static_assert(TK % Op::kK == 0, "stage depth");

    __shared__ __attribute__((aligned(16))) bf16_t As[2][TM][LD];
    __shared__ __attribute__((aligned(16))) bf16_t Bs[2][TN][LD];

    const int kh = p.kh, kw = p.kw;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave % WM;
    const int wn = wave / WM;
    // XCD-contiguous tile order, row tiles fastest (as in the fp32 kernel)
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
    const int M = p.M, Rp = p.Rp;
    const int IH = p.IH, IW = p.IW, Ctot = p.Ctot;
    const int OHW = p.OH * p.OW;
    const int Cg8 = p.Cgp >> 3;

    const __amdgpu_buffer_rsrc_t ra = make_rsrc(p.A, p.A_bytes);
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(p.X, p.X_bytes);

    // ---- B: one output column per thread; its chunk slots are wave-uniform
    const int bcl = tid % TN;
    const int slot0 = __builtin_amdgcn_readfirstlane(tid / TN);
    int b_ih0, b_iw0, b_base;
    uint32_t b_cbad;
    {
        const int col = n0 + bcl;
        const int n = col / OHW;
        const int pix = col - n * OHW;
        const int i = pix / p.OW;
        const int j = pix - i * p.OW;
        b_ih0 = i * p.sh - p.ph;
        b_iw0 = j * p.sw - p.pw;
        b_base = ((n * IH + b_ih0) * IW + b_iw0) * Ctot + g * p.Cgp;
        b_cbad = (uint32_t)(col >= p.Ncol) << 31;
    }
    // Reduction walk of each slot: chunk kc = s*TB + slot0 + BS*q sits at tap
    // (wu, wv), channels 8*wc .. 8*wc + 7.  Scalar state, advanced by TB
    // chunks per stage.
    int wu[EB], wv[EB], wc[EB];
#pragma unroll
    for (int q = 0; q < EB; ++q) {
        const int kc = slot0 + BS * q;
        const int t = kc / Cg8;
        wc[q] = kc - t * Cg8;
        wu[q] = t / kw;
        wv[q] = t - wu[q] * kw;
    }
    auto advance = [&]() {
#pragma unroll
        for (int q = 0; q < EB; ++q) {
            wc[q] += TB;
            while (wc[q] >= Cg8) {
                wc[q] -= Cg8;
                if (++wv[q] == kw) {
                    wv[q] = 0;
                    ++wu[q];
                }
            }
        }
    };

    u32x4 rA[EA], rB[EB];
    auto load_a = [&](int kbase) {
#pragma unroll
        for (int q = 0; q < EA; ++q) {
            const int id = tid + NT * q;
            const int row = id / TB;
            const int kc = id % TB;
            const uint32_t bad = ((uint32_t)(id >= CA) | (uint32_t)(m0 + row >= M)) << 31;
            rA[q] = buf_ld_b128(ra, ((uint32_t)((g * M + m0 + row) * Rp + kbase + kc * 8) * 2u) |
                                        bad);
        }
    };
    auto load_b = [&]() {
#pragma unroll
        for (int q = 0; q < EB; ++q) {
            const int delta = (wu[q] * IW + wv[q]) * Ctot + wc[q] * 8;
            const int ih = b_ih0 + wu[q];
            const int iw = b_iw0 + wv[q];
            const uint32_t bad = ((uint32_t)(wu[q] >= kh) |
                                  (uint32_t)((unsigned)ih >= (unsigned)IH) |
                                  (uint32_t)((unsigned)iw >= (unsigned)IW)) << 31;
            rB[q] = buf_ld_b128(rx, ((uint32_t)(b_base + delta) * 2u) | bad | b_cbad);
        }
    };
    auto store_stage = [&](int buf) {
#pragma unroll
        for (int q = 0; q < EA; ++q) {
            const int id = tid + NT * q;
            if (CA % NT == 0 || id < CA)
                *(u32x4*)&As[buf][id / TB][(id % TB) * 8] = rA[q];
        }
#pragma unroll
        for (int q = 0; q < EB; ++q)
            *(u32x4*)&Bs[buf][bcl][(slot0 + BS * q) * 8] = rB[q];
    };

    // forward: accumulators start at the bias of their row
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

    const int nst = Rp / TK;
    load_a(0);
    load_b();
    store_stage(0);
    __syncthreads();

    const int arow = wm * MI * MT + lane % MT;
    const int brow = wn * NI * MT + lane % MT;
    const int kl = (lane / MT) * 8;

    for (int s = 0; s < nst; ++s) {
        const int cur = s & 1;
        if (s + 1 < nst) {
            load_a((s + 1) * TK);
            advance();
            load_b();
        }
        constexpr int PF = KS > 1 ? 1 : 0;
        bf16x8 fa[PF + 1][MI], fb[PF + 1][NI];
        auto read_frag = [&](int ks, int slot) {
#pragma unroll
            for (int mi = 0; mi < MI; ++mi)
                fa[slot][mi] = lds_frag(&As[cur][arow + mi * MT][ks * Op::kK + kl]);
#pragma unroll
            for (int ni = 0; ni < NI; ++ni)
                fb[slot][ni] = lds_frag(&Bs[cur][brow + ni * MT][ks * Op::kK + kl]);
        };
        read_frag(0, 0);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            if (ks + PF < KS && PF > 0)
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
    if constexpr (EPI == 0) {
        int cbase[NI];
        uint32_t cbad[NI];
#pragma unroll
        for (int ni = 0; ni < NI; ++ni) {
            const int col = n0 + brow + ni * MT;
            const int n = col / OHW;
            const int pix = col - n * OHW;
            cbase[ni] = n * p.Cout * OHW + pix;
            cbad[ni] = (uint32_t)(col >= p.Ncol) << 31;
        }
#pragma unroll
        for (int mi = 0; mi < MI; ++mi) {
#pragma unroll
            for (int ni = 0; ni < NI; ++ni) {
#pragma unroll
                for (int q = 0; q < Op::kRegs; ++q) {
                    const int m = m0 + wm * MI * MT + mi * MT + Op::row(q, lane);
                    const int oc = g * M + m;
                    const float z = acc[mi][ni][q];
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
        const __amdgpu_buffer_rsrc_t rom = make_rsrc(p.Omask, MASK ? p.Y_bytes / 2 : 0u);
        int cb[NI], hb[NI], wb[NI];
#pragma unroll
        for (int ni = 0; ni < NI; ++ni) {
            const int col = n0 + brow + ni * MT;
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
                    const uint32_t idx = (uint32_t)(cb[ni] + c * OutHW + h * p.OutW + w);
                    float v = acc[mi][ni][q];
                    if constexpr (MASK) {
                        // backward of the ReLU whose (bf16) output is this
                        // layer's bottom: keep the gradient where it was > 0
                        const float y = bf16_to_f32(buf_ld_u16(rom, (idx * 2u) | bad));
                        v = y > 0.f ? v : 0.f;
                    }
                    buf_st_f32(v, ry, (idx * 4u) | bad);
                }
            }
        }
    }
}

// ----------------------------------------------------------- weight gradient
// Split-K over the output pixels (n, i, j), 32 per stage.  Both operands are
// gathered as 16-byte chunks of 8 channels per pixel; each thread loads the
// same chunk row for two adjacent pixels and writes the pair of values of
// every channel as one 32-bit word, so LDS rows hold consecutive pixels (the
// reduction index) as the bf16 instructions want them.
template <int WM, int WN, int MI, int NI>
__global__ void __launch_bounds__(64 * WM * WN)
conv_wgrad_bf16_kernel(const WgradBf16Params p)
{
    constexpr int MT = 32;
    constexpr int NT = 64 * WM * WN;
    constexpr int TM = WM * MI * MT;
    constexpr int TN = WN * NI * MT;
    constexpr int TKP = 32;            // pixels per stage
    constexpr int PP = TKP / 2;        // pixel pairs per stage
    constexpr int LD = TKP + 8;
    constexpr int RS = NT / PP;        // chunk rows covered by one pass
    constexpr int CAM = TM / 8, CBN = TN / 8;
    constexpr int EA = (CAM + RS - 1) / RS;
    constexpr int EB = (CBN + RS - 1) / RS;
    constexpr int KS = TKP / 16;

    __shared__ __attribute__((aligned(16))) bf16_t As[2][TM][LD];
    __shared__ __attribute__((aligned(16))) bf16_t Bs[2][TN][LD];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave % WM;
    const int wn = wave / WM;
    const int n_rt = (p.Rw + TN - 1) / TN;
    const int n_mt = (p.Kg + TM - 1) / TM;
    const int T = blockIdx.x;
    if (T >= n_rt * n_mt * p.G * p.splits)
        return;
    const int rt = T % n_rt;
    const int mt = (T / n_rt) % n_mt;
    const int g = (T / (n_rt * n_mt)) % p.G;
    const int split = T / (n_rt * n_mt * p.G);
    const int m0 = mt * TM;
    const int r0 = rt * TN;
    const int IH = p.IH, IW = p.IW, Ctot = p.Ctot;
    const int OHW = p.OH * p.OW;
    const int col_begin = split * p.cols_per_split;
    const int col_end = min(p.Ncol, col_begin + p.cols_per_split);

    const __amdgpu_buffer_rsrc_t rd = make_rsrc(p.D, p.D_bytes);
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(p.X, p.X_bytes);

    const int pp = tid % PP;  // pixel pair within a stage
    const int cr = tid / PP;  // chunk row within a pass

    // A chunk rows: channels m0 + 8*(cr + RS*q) .. +7 of the group
    int a_off[EA];
    uint32_t a_bad[EA];
#pragma unroll
    for (int q = 0; q < EA; ++q) {
        const int row = cr + RS * q;
        a_off[q] = g * p.Kgp + m0 + 8 * row;
        a_bad[q] = ((uint32_t)(row >= CAM) | (uint32_t)(m0 + 8 * row >= p.Kg)) << 31;
    }
    // B chunk rows: r = r0 + 8*(cr + RS*q) = (u, v, c) over kh x kw x Cgp
    int b_u[EB], b_v[EB], b_off[EB];
    uint32_t b_bad[EB];
#pragma unroll
    for (int q = 0; q < EB; ++q) {
        const int row = cr + RS * q;
        const int r = r0 + 8 * row;
        const int t = r / p.Cgp;
        const int c = r - t * p.Cgp;
        b_u[q] = t / p.kw;
        b_v[q] = t - b_u[q] * p.kw;
        b_off[q] = (b_u[q] * IW + b_v[q]) * Ctot + g * p.Cgp + c;
        b_bad[q] = ((uint32_t)(row >= CBN) | (uint32_t)(r >= p.Rw)) << 31;
    }

    u32x4 rA[EA][2], rB[EB][2];
    auto load_stage = [&](int cbase) {
#pragma unroll
        for (int e = 0; e < 2; ++e) {
            const int col = cbase + 2 * pp + e;
            const uint32_t cbad = (uint32_t)(col >= col_end) << 31;
            const int n = (int)fdiv((uint32_t)col, p.div_ohw);
            const int pix = col - n * OHW;
            const int i = (int)fdiv((uint32_t)pix, p.div_ow);
            const int j = pix - i * p.OW;
            const int ih0 = i * p.sh - p.ph;
            const int iw0 = j * p.sw - p.pw;
            const int xbase = ((n * IH + ih0) * IW + iw0) * Ctot;
#pragma unroll
            for (int q = 0; q < EA; ++q)
                rA[q][e] = buf_ld_b128(
                    rd, ((uint32_t)(col * p.Ktot + a_off[q]) * 2u) | cbad | a_bad[q]);
#pragma unroll
            for (int q = 0; q < EB; ++q) {
                const int ih = ih0 + b_u[q];
                const int iw = iw0 + b_v[q];
                const uint32_t bad = ((uint32_t)((unsigned)ih >= (unsigned)IH) |
                                      (uint32_t)((unsigned)iw >= (unsigned)IW)) << 31;
                rB[q][e] = buf_ld_b128(
                    rx, ((uint32_t)(xbase + b_off[q]) * 2u) | cbad | bad | b_bad[q]);
            }
        }
    };
    // channel k of the two pixels -> one word (pixel 2pp in the low half)
    auto pair = [](const u32x4& x0, const u32x4& x1, int k) -> uint32_t {
        const uint32_t w0 = x0[k >> 1], w1 = x1[k >> 1];
        return (k & 1) ? ((w0 >> 16) | (w1 & 0xffff0000u)) : ((w0 & 0xffffu) | (w1 << 16));
    };
    auto store_stage = [&](int buf) {
#pragma unroll
        for (int q = 0; q < EA; ++q) {
            const int row = cr + RS * q;
            if (CAM % RS == 0 || row < CAM) {
#pragma unroll
                for (int k = 0; k < 8; ++k)
                    *(uint32_t*)&As[buf][8 * row + k][2 * pp] = pair(rA[q][0], rA[q][1], k);
            }
        }
#pragma unroll
        for (int q = 0; q < EB; ++q) {
            const int row = cr + RS * q;
            if (CBN % RS == 0 || row < CBN) {
#pragma unroll
                for (int k = 0; k < 8; ++k)
                    *(uint32_t*)&Bs[buf][8 * row + k][2 * pp] = pair(rB[q][0], rB[q][1], k);
            }
        }
    };

    floatx16 acc[MI][NI];
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int ni = 0; ni < NI; ++ni)
            acc[mi][ni] = floatx16{};

    const int nst = col_end > col_begin ? (col_end - col_begin + TKP - 1) / TKP : 0;
    if (nst > 0) {
        load_stage(col_begin);
        store_stage(0);
    }
    __syncthreads();

    const int arow = wm * MI * MT + (lane & 31);
    const int brow = wn * NI * MT + (lane & 31);
    const int kl = (lane >> 5) * 8;

    for (int s = 0; s < nst; ++s) {
        const int cur = s & 1;
        if (s + 1 < nst)
            load_stage(col_begin + (s + 1) * TKP);
        bf16x8 fa[KS][MI], fb[KS][NI];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
            for (int mi = 0; mi < MI; ++mi)
                fa[ks][mi] = lds_frag(&As[cur][arow + mi * MT][ks * 16 + kl]);
#pragma unroll
            for (int ni = 0; ni < NI; ++ni)
                fb[ks][ni] = lds_frag(&Bs[cur][brow + ni * MT][ks * 16 + kl]);
        }
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
            for (int mi = 0; mi < MI; ++mi)
#pragma unroll
                for (int ni = 0; ni < NI; ++ni)
                    acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[ks][mi], fb[ks][ni],
                                                                        acc[mi][ni], 0, 0, 0);
        if (s + 1 < nst)
            store_stage(cur ^ 1);
        __syncthreads();
    }

    // Partial result P[split][g*Kg + m][r], r = (u, v, c) over Rw (lanes along r)
    const __amdgpu_buffer_rsrc_t rp = make_rsrc(p.P, p.P_bytes);
    const int pbase = split * p.K * p.Rw;
#pragma unroll
    for (int ni = 0; ni < NI; ++ni) {
        const int r = r0 + brow + ni * MT;
#pragma unroll
        for (int mi = 0; mi < MI; ++mi) {
#pragma unroll
            for (int q = 0; q < 16; ++q) {
                const int m = m0 + wm * MI * MT + mi * MT + 8 * (q >> 2) + 4 * (lane >> 5) + (q & 3);
                const uint32_t bad = ((uint32_t)(m >= p.Kg) | (uint32_t)(r >= p.Rw)) << 31;
                buf_st_f32(acc[mi][ni][q], rp,
                           ((uint32_t)(pbase + (g * p.Kg + m) * p.Rw + r) * 4u) | bad);
            }
        }
    }
}

// dW[k][c][t] = (accumulate ? dW : 0) + sum_s P[s][k][t*Cgp + c]  (c < Cg, t < khw):
// the split partials added in a fixed order, as wgrad_reduce_kernel does, with
// lanes along the partials' (u, v, c) order.
constexpr int kPermParts = 8;
constexpr int kPermCols = 32;

__global__ void __launch_bounds__(kPermParts * kPermCols)
wgrad_reduce_perm_kernel(const float* __restrict__ P, float* __restrict__ dW, int K, int Rw,
                         int Cgp, int Cg, int khw, int splits, int accumulate)
{
    __shared__ float part[kPermParts][kPermCols + 1];
    const int col = threadIdx.x % kPermCols;
    const int pt = threadIdx.x / kPermCols;
    const int count = K * Rw;
    const int e = blockIdx.x * kPermCols + col;
    float s = 0.f;
    if (e < count) {
        int q = pt;
        for (; q + 3 * kPermParts < splits; q += 4 * kPermParts) {
            const float a0 = P[(size_t)q * count + e];
            const float a1 = P[(size_t)(q + kPermParts) * count + e];
            const float a2 = P[(size_t)(q + 2 * kPermParts) * count + e];
            const float a3 = P[(size_t)(q + 3 * kPermParts) * count + e];
            s += a0;
            s += a1;
            s += a2;
            s += a3;
        }
        for (; q < splits; q += kPermParts)
            s += P[(size_t)q * count + e];
    }
    part[pt][col] = s;
    __syncthreads();
    if (pt == 0 && e < count) {
        float t = 0.f;
#pragma unroll
        for (int i = 0; i < kPermParts; ++i)
            t += part[i][col];
        const int k = e / Rw;
        const int r = e - k * Rw;
        const int tap = r / Cgp;
        const int c = r - tap * Cgp;
        if (c < Cg && tap < khw) {
            float* o = dW + ((size_t)k * Cg + c) * khw + tap;
            *o = accumulate ? *o + t : t;
        }
    }
}

// ------------------------------------------------------------------ staging
// NCHW bf16 -> channel-contiguous bf16 with per-group channel padding, through
// a CT-channel x (4096/CT)-pixel LDS tile (CT = 8 .. 64, sized to the padded
// channel count): coalesced 2-byte reads along pixels, 16-byte writes along
// channels.
template <int CT>
__global__ void __launch_bounds__(256)
nhwc_from_nchw_bf16_kernel(const bf16_t* __restrict__ X, bf16_t* __restrict__ Xh, int C, int HW,
                           int Cg, int Cgp, int Ctot, int ptiles, int ctiles)
{
    constexpr int PT = 4096 / CT;
    constexpr int C8 = CT / 8;
    __shared__ bf16_t tile[CT][PT + 2];
    // block -> (n, channel tile, pixel tile), pixel tiles fastest
    const int n = blockIdx.x / (ptiles * ctiles);
    const int rem = blockIdx.x - n * ptiles * ctiles;
    const int ct = rem / ptiles;
    const int c0 = ct * CT;
    const int p0 = (rem - ct * ptiles) * PT;
    const int tid = threadIdx.x;
#pragma unroll 4
    for (int q = 0; q < 16; ++q) {
        const int e = tid + 256 * q;
        const int c = e / PT;
        const int px = e % PT;
        const int cp = c0 + c;
        const int g = cp / Cgp;
        const int cl = cp - g * Cgp;
        const int pix = p0 + px;
        bf16_t v = 0;
        if (cp < Ctot && cl < Cg && pix < HW)
            v = X[((size_t)n * C + g * Cg + cl) * HW + pix];
        tile[c][px] = v;
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < 2; ++q) {
        const int id = tid + 256 * q;
        const int px = id / C8;
        const int c8 = id % C8;
        const int pix = p0 + px;
        const int cp = c0 + 8 * c8;
        if (pix < HW && cp < Ctot) {
            u32x4 w;
#pragma unroll
            for (int k = 0; k < 4; ++k)
                w[k] = (uint32_t)tile[8 * c8 + 2 * k][px] |
                       ((uint32_t)tile[8 * c8 + 2 * k + 1][px] << 16);
            *(u32x4*)&Xh[((size_t)n * HW + pix) * Ctot + cp] = w;
        }
    }
}

// Top-gradient staging: Dh = bf16(relu ? G [Y > 0] : G) channel-contiguous,
// one block per (image, 64 padded channels, 64 pixels).  Each wave also sums
// the fp32 masked gradient of its channels over the block's pixels (a fixed
// butterfly) into sums[(g*Kg + k) * T + n * ptiles + pt]: the bias-gradient
// partials, T = N * ptiles per channel.
__global__ void __launch_bounds__(256)
diff_prep_bf16_kernel(const float* __restrict__ G, const float* __restrict__ Y,
                      bf16_t* __restrict__ Dh, float* __restrict__ sums, int K, int HW, int Kg,
                      int Kgp, int Ktot, int relu, int ptiles, int ctiles, int T)
{
    __shared__ bf16_t tile[64][66];
    const int n = blockIdx.x / (ptiles * ctiles);
    const int rem = blockIdx.x - n * ptiles * ctiles;
    const int ct = rem / ptiles;
    const int pt = rem - ct * ptiles;
    const int c0 = ct * 64;
    const int p0 = pt * 64;
    const int tid = threadIdx.x;
    const int px = tid & 63;
    const int cw = tid >> 6;
    const int pix = p0 + px;
#pragma unroll 4
    for (int q = 0; q < 16; ++q) {
        const int cl = cw + 4 * q;
        const int cp = c0 + cl;
        const int g = cp / Kgp;
        const int k = cp - g * Kgp;
        const bool ok = cp < Ktot && k < Kg;
        float d = 0.f;
        if (ok && pix < HW) {
            const size_t idx = ((size_t)n * K + g * Kg + k) * HW + pix;
            d = G[idx];
            if (relu && !(Y[idx] > 0.f))
                d = 0.f;
        }
        tile[cl][px] = f32_to_bf16_rne(d);
        if (sums) {
            const float s = wave_sum(d);
            if (px == 0 && ok)
                sums[(size_t)(g * Kg + k) * T + n * ptiles + pt] = s;
        }
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < 2; ++q) {
        const int id = tid + 256 * q;
        const int pl = id >> 3;
        const int c8 = id & 7;
        const int pw = p0 + pl;
        const int cp = c0 + 8 * c8;
        if (pw < HW && cp < Ktot) {
            u32x4 w;
#pragma unroll
            for (int k = 0; k < 4; ++k)
                w[k] = (uint32_t)tile[8 * c8 + 2 * k][pl] |
                       ((uint32_t)tile[8 * c8 + 2 * k + 1][pl] << 16);
            *(u32x4*)&Dh[((size_t)n * HW + pw) * Ktot + cp] = w;
        }
    }
}

// db[k] = (accumulate ? db[k] : 0) + sum_{t < T} sums[k*T + t]: one block per
// channel, thread i adds the terms i, i + 256, ... in order, then a fixed
// pairwise tree over the threads.
__global__ void __launch_bounds__(256)
bias_reduce_kernel(const float* __restrict__ sums, float* __restrict__ db, int T, int accumulate)
{
    __shared__ float red[256];
    const int k = blockIdx.x;
    const float* src = sums + (size_t)k * T;
    float s = 0.f;
    for (int t = threadIdx.x; t < T; t += 256)
        s += src[t];
    red[threadIdx.x] = s;
    __syncthreads();
    for (int off = 128; off > 0; off >>= 1) {
        if (threadIdx.x < off)
            red[threadIdx.x] += red[threadIdx.x + off];
        __syncthreads();
    }
    if (threadIdx.x == 0)
        db[k] = accumulate ? db[k] + red[0] : red[0];
}

// Forward weights: Wp[o][(u*kw + v)*Cgp + c] = W[o][c][u][v], zero for c >= Cg
// and for r >= khw*Cgp (rows padded to Rp).
__global__ void __launch_bounds__(256)
pack_weights_bf16_kernel(const bf16_t* __restrict__ W, bf16_t* __restrict__ Wp, int K, int Cg,
                         int Cgp, int khw, int Rp)
{
    const long total = (long)K * Rp;
    for (long e = blockIdx.x * (long)blockDim.x + threadIdx.x; e < total;
         e += (long)gridDim.x * blockDim.x) {
        const int o = (int)(e / Rp);
        const int r = (int)(e - (long)o * Rp);
        const int t = r / Cgp;
        const int c = r - t * Cgp;
        bf16_t v = 0;
        if (t < khw && c < Cg)
            v = W[((long)o * Cg + c) * khw + t];
        Wp[e] = v;
    }
}

// Phase-stacked data-gradient weights (as dgrad_weight_transform_kernel) with
// the reduction index tap-major over padded channels:
// Wt[g][m = (c, fh, fw)][(th*Tw + tw)*Kgp + k] = W[g*Kg + k][c][fh + sh*(Th-1-th)][fw + sw*(Tw-1-tw)],
// zero past the kernel edge, for k >= Kg and for r >= Th*Tw*Kgp (rows padded to Rtp).
__global__ void __launch_bounds__(256)
dgrad_weights_bf16_kernel(const bf16_t* __restrict__ W, bf16_t* __restrict__ Wt, int G, int Kg,
                          int Kgp, int Cg, int kh, int kw, int sh, int sw, int Th, int Tw, int Rtp)
{
    const int Mt = Cg * sh * sw;
    const long total = (long)G * Mt * Rtp;
    for (long e = blockIdx.x * (long)blockDim.x + threadIdx.x; e < total;
         e += (long)gridDim.x * blockDim.x) {
        const int r = (int)(e % Rtp);
        const long gm = e / Rtp;
        const int m = (int)(gm % Mt);
        const int g = (int)(gm / Mt);
        const int t = r / Kgp;
        const int k = r - t * Kgp;
        bf16_t v = 0;
        if (t < Th * Tw && k < Kg) {
            const int th = t / Tw, tw = t - th * Tw;
            const int c = m / (sh * sw);
            const int f = m - c * sh * sw;
            const int fh = f / sw, fw = f - fh * sw;
            const int u = fh + sh * (Th - 1 - th);
            const int v2 = fw + sw * (Tw - 1 - tw);
            if (u < kh && v2 < kw)
                v = W[(((long)(g * Kg + k) * Cg + c) * kh + u) * kw + v2];
        }
        Wt[e] = v;
    }
}

// ------------------------------------------------------------------ launch
namespace {

unsigned grid_1d(long total)
{
    long blocks = (total + 255) / 256;
    return (unsigned)(blocks > 4096 ? 4096 : (blocks < 1 ? 1 : blocks));
}

template <int MT, int WM, int WN, int MI, int NI, int TK, int EPI, bool MASK>
hipError_t launch_gemm(const GemmBf16Params& p, hipStream_t s)
{
    constexpr int TM = WM * MI * MT, TN = WN * NI * MT;
    const int64_t tiles = (int64_t)((p.Ncol + TN - 1) / TN) * ((p.M + TM - 1) / TM) * p.G;
    const int64_t per_xcd = (tiles + 7) / 8;
    hipLaunchKernelGGL((conv_gemm_bf16_kernel<MT, WM, WN, MI, NI, TK, EPI, MASK>),
                       dim3((unsigned)(per_xcd * 8)), dim3(64 * WM * WN), 0, s, p);
    return hipGetLastError();
}

template <int EPI, bool MASK>
hipError_t launch_gemm_tile(const GemmBf16Params& p, int tile, hipStream_t s)
{
    switch (tile) {
    case TILE_128x128:
        return launch_gemm<32, 2, 2, 2, 2, kBf16TK, EPI, MASK>(p, s);
    case TILE_96x256:
        return launch_gemm<32, 1, 4, 3, 2, kBf16TK, EPI, MASK>(p, s);
    case TILE_48x256:
        return launch_gemm<16, 1, 4, 3, 4, kBf16TK, EPI, MASK>(p, s);
    case TILE_64x256:
        return launch_gemm<32, 1, 4, 2, 2, kBf16TK, EPI, MASK>(p, s);
    default:
        return hipErrorInvalidValue;
    }
}

template <int WM, int WN, int MI, int NI>
hipError_t launch_wg(const WgradBf16Params& p, hipStream_t s)
{
    constexpr int TM = WM * MI * 32, TN = WN * NI * 32;
    const int64_t tiles = (int64_t)((p.Rw + TN - 1) / TN) * ((p.Kg + TM - 1) / TM) * p.G * p.splits;
    hipLaunchKernelGGL((conv_wgrad_bf16_kernel<WM, WN, MI, NI>), dim3((unsigned)tiles),
                       dim3(64 * WM * WN), 0, s, p);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_conv_gemm_bf16(const GemmBf16Params& p, int epi, int tile, hipStream_t s)
{
    if (p.Ncol == 0)
        return hipSuccess;
    if (p.Rp % kBf16TK != 0 || p.Cgp % 8 != 0 || p.Ctot % 8 != 0)
        return hipErrorInvalidValue;
    if (epi == 0)
        return launch_gemm_tile<0, false>(p, tile, s);
    return p.Omask ? launch_gemm_tile<1, true>(p, tile, s) : launch_gemm_tile<1, false>(p, tile, s);
}

hipError_t launch_conv_wgrad_bf16(const WgradBf16Params& p, int tile, hipStream_t s)
{
    if (p.Cgp % 8 != 0 || p.Kgp % 8 != 0)
        return hipErrorInvalidValue;
    switch (tile) {
    case WTILE_128x128:
        return launch_wg<2, 2, 2, 2>(p, s);
    case WTILE_96x128:
        return launch_wg<1, 4, 3, 1>(p, s);
    case WTILE_64x128:
        return launch_wg<2, 2, 1, 2>(p, s);
    default:
        return hipErrorInvalidValue;
    }
}

hipError_t launch_wgrad_reduce_perm(const float* P, float* dW, int K, int Rw, int Cgp, int Cg,
                                    int khw, int splits, int accumulate, hipStream_t s)
{
    const int count = K * Rw;
    if (count == 0)
        return hipSuccess;
    hipLaunchKernelGGL(wgrad_reduce_perm_kernel, dim3((count + kPermCols - 1) / kPermCols),
                       dim3(kPermParts * kPermCols), 0, s, P, dW, K, Rw, Cgp, Cg, khw, splits,
                       accumulate);
    return hipGetLastError();
}

hipError_t launch_nhwc_from_nchw_bf16(const uint16_t* X, uint16_t* Xh, int N, int C, int HW,
                                      int Cg, int Cgp, int Ctot, hipStream_t s)
{
    if (N == 0)
        return hipSuccess;
    const int ct = Ctot <= 8 ? 8 : Ctot <= 16 ? 16 : Ctot <= 32 ? 32 : 64;
    const int pt = 4096 / ct;
    const int ptiles = (HW + pt - 1) / pt;
    const int ctiles = (Ctot + ct - 1) / ct;
    const dim3 grid((unsigned)((int64_t)ptiles * ctiles * N));
    switch (ct) {
    case 8:
        hipLaunchKernelGGL(nhwc_from_nchw_bf16_kernel<8>, grid, dim3(256), 0, s, X, Xh, C, HW, Cg,
                           Cgp, Ctot, ptiles, ctiles);
        break;
    case 16:
        hipLaunchKernelGGL(nhwc_from_nchw_bf16_kernel<16>, grid, dim3(256), 0, s, X, Xh, C, HW, Cg,
                           Cgp, Ctot, ptiles, ctiles);
        break;
    case 32:
        hipLaunchKernelGGL(nhwc_from_nchw_bf16_kernel<32>, grid, dim3(256), 0, s, X, Xh, C, HW, Cg,
                           Cgp, Ctot, ptiles, ctiles);
        break;
    default:
        hipLaunchKernelGGL(nhwc_from_nchw_bf16_kernel<64>, grid, dim3(256), 0, s, X, Xh, C, HW, Cg,
                           Cgp, Ctot, ptiles, ctiles);
        break;
    }
    return hipGetLastError();
}

int diff_prep_terms(int N, int HW) { return N * ((HW + 63) / 64); }

hipError_t launch_diff_prep_bf16(const float* G, const float* Y, uint16_t* Dh, float* sums, int N,
                                 int K, int HW, int Kg, int Kgp, int Ktot, int relu, hipStream_t s)
{
    if (N == 0)
        return hipSuccess;
    const int ptiles = (HW + 63) / 64;
    const int ctiles = (Ktot + 63) / 64;
    hipLaunchKernelGGL(diff_prep_bf16_kernel, dim3((unsigned)((int64_t)ptiles * ctiles * N)),
                       dim3(256), 0, s, G, Y, Dh, sums, K, HW, Kg, Kgp, Ktot, relu, ptiles, ctiles,
                       N * ptiles);
    return hipGetLastError();
}

hipError_t launch_bias_reduce(const float* sums, float* db, int T, int K, int accumulate,
                              hipStream_t s)
{
    if (K == 0)
        return hipSuccess;
    hipLaunchKernelGGL(bias_reduce_kernel, dim3(K), dim3(256), 0, s, sums, db, T, accumulate);
    return hipGetLastError();
}

hipError_t launch_pack_weights_bf16(const uint16_t* W, uint16_t* Wp, int K, int Cg, int Cgp,
                                    int khw, int Rp, hipStream_t s)
{
    const long total = (long)K * Rp;
    if (total == 0)
        return hipSuccess;
    hipLaunchKernelGGL(pack_weights_bf16_kernel, dim3(grid_1d(total)), dim3(256), 0, s, W, Wp, K,
                       Cg, Cgp, khw, Rp);
    return hipGetLastError();
}

hipError_t launch_dgrad_weights_bf16(const uint16_t* W, uint16_t* Wt, int G, int Kg, int Kgp,
                                     int Cg, int kh, int kw, int sh, int sw, int Th, int Tw,
                                     int Rtp, hipStream_t s)
{
    const long total = (long)G * Cg * sh * sw * Rtp;
    if (total == 0)
        return hipSuccess;
    hipLaunchKernelGGL(dgrad_weights_bf16_kernel, dim3(grid_1d(total)), dim3(256), 0, s, W, Wt, G,
                       Kg, Kgp, Cg, kh, kw, sh, sw, Th, Tw, Rtp);
    return hipGetLastError();
}

}  // namespace caffe_hip
