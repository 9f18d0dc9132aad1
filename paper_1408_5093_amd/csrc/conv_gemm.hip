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

// One wave copies 64 consecutive floats into LDS at `dst` (wave-uniform):
// lane i's element from byte offset voff + soff lands at dst + 4*i.  An offset
// with bit 31 set is out of range and writes 0.
__device__ __forceinline__ void copy_to_lds(__amdgpu_buffer_rsrc_t r, float* dst, uint32_t voff,
                                            uint32_t soff)
{
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)dst, 4, voff, soff, 0, 0);
}

template <int MT, int WM, int WN, int MI, int NI, int TK, int KH, int KW, int SH, int SW, int EPI,
          bool TAP, bool MASK>
__global__ void __launch_bounds__(64 * WM * WN)
conv_gemm_f32_kernel(const ConvGemmParams p)
{
    typedef Mfma<MT> Op;
    constexpr int NT = 64 * WM * WN;
    constexpr int NW = NT / 64;          // waves
    constexpr int TM = WM * MI * MT;
    constexpr int TN = WN * NI * MT;
    constexpr int KS = TK / Op::kStep;
    constexpr int NC = TN / 64;          // 64-column copies per B row of the tile
    constexpr int NA = TK * TM / 64 / NW;  // A copies per wave per stage
    constexpr int NB = TK * NC / NW;       // B copies per wave per stage
    static_assert(TN % 64 == 0 && NW % NC == 0, "B copy mapping");
    static_assert(TK * TM % (64 * NW) == 0 && TK * NC % NW == 0, "copy split");
    static_assert(TK % Op::kStep == 0, "stage depth");
    // A is staged as the flat [TK][TM] array (row stride TM: 96 and 48 put the
    // k rows a fragment read touches on distinct banks); B rows hold whole
    // 64-column copies, with a stride of 16 (mod 32) for the 16x16x4
    // fragments, which read four k rows at once.
    constexpr int LDA = TM;
    constexpr int LDB = TN + (MT == 16 ? 16 : 0);

    // One array per pipeline buffer: with the buffer a compile-time choice
    // (the stage loop below is unrolled by two), the compiler can tell the
    // copies into one buffer from the fragment reads of the other and inserts
    // no waits between them.
    __shared__ float As0[TK][LDA], As1[TK][LDA];
    __shared__ float Bs0[TK][LDB], Bs1[TK][LDB];
    typedef float ATile[TK][LDA];
    typedef float BTile[TK][LDB];

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
    const int n_tiles = n_mt * n_ct * p.G;
    const bool has_tail = EPI < 2 && p.tail_splits > 1;
    int T = blockIdx.x;
    if (p.xcd_order) {
        const int x = blockIdx.x & 7, i = blockIdx.x >> 3;
        if (has_tail) {
            // each XCD takes a contiguous run of the whole tiles, then an
            // eighth of the tail's work items, which fill its units last
            const int n_items = (n_tiles - p.tail_T) * p.tail_splits;
            const int fq = (p.tail_T + 7) >> 3, tq = (n_items + 7) >> 3;
            if (i < fq) {
                const int f = x * fq + i;
                T = f < p.tail_T ? f : INT_MAX;
            } else {
                const int j = x * tq + (i - fq);
                T = j < n_items ? p.tail_T + j : INT_MAX;
            }
        } else {
            T = x * (int)(gridDim.x >> 3) + i;
        }
    }
    // EPI 2 (dense) and EPI 3 (gathered convolution operands) store split-K
    // partials: the reduction is cut into p.splits ranges of
    // p.stages_per_split stages, the split index varying slowest.  EPI 0 and
    // 1 may cut only their last tiles (a tail split, see ConvGemmParams):
    // work item T >= tail_T takes reduction range (T - tail_T) % tail_splits
    // of tile tail_T + (T - tail_T) / tail_splits.
    int tile = T, split = 0;
    bool tail = false;
    if constexpr (EPI >= 2) {
        if (T >= n_tiles * p.splits)
            return;
        tile = T % n_tiles;
        split = T / n_tiles;
    } else {
        if (has_tail && T >= p.tail_T) {
            const int j = T - p.tail_T;
            const int jt = j / p.tail_splits;
            tile = p.tail_T + jt;
            split = j - jt * p.tail_splits;
            tail = true;
        }
        if (tile >= n_tiles)
            return;
    }
    const int mt = tile % n_mt;
    const int ct = (tile / n_mt) % n_ct;
    const int g = tile / (n_mt * n_ct);
    const int m0 = mt * TM;
    const int n0 = ct * TN;
    const int M = p.M, R = p.R;
    const int IH = p.IH, IW = p.IW, IHW = IH * IW;
    const int OHW = p.OH * p.OW;
    const int Cin_g = p.Cin_g;

    const __amdgpu_buffer_rsrc_t ra = make_rsrc(p.A, p.A_bytes);
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(p.X, p.X_bytes);

    // Operands go from global memory straight to LDS, one wave copy = 64
    // consecutive floats.  A copy j of a stage (j = wave + NW*q) covers the
    // flat elements 64*j .. 64*j + 63 of the [TK][TM] A tile: lane l takes
    // k row (64*j + l) / TM, tile row (64*j + l) % TM of A (laid out
    // [group][r][m], m contiguous); its offset without the stage's k base is
    // fixed for the kernel.  B copy j covers k row j / NC, columns
    // n0 + 64*(j % NC) + lane; a wave's column is fixed and its k rows advance
    // by NW / NC per copy.
    // A rows past M need no mask: they only feed accumulator rows the
    // epilogue never stores, and their loads stay inside A or read 0.
    // (When TM is a multiple of 64 a copy's k row and column offset are
    // wave-uniform and go to the scalar offset; one lane offset serves all.)
    constexpr bool A_UNIFORM = TM % 64 == 0;
    uint32_t a_voff[A_UNIFORM ? 1 : NA];
    int a_k[A_UNIFORM ? 1 : NA];  // the lane's k row within a stage, per copy
#pragma unroll
    for (int q = 0; q < (A_UNIFORM ? 1 : NA); ++q) {
        const int flat = A_UNIFORM ? lane : 64 * (wave + NW * q) + lane;
        const int k = flat / TM;
        a_k[q] = k;
        a_voff[q] = (uint32_t)((g * R + k) * M + m0 + flat - k * TM) * 4u;
    }
    const uint32_t a_row4 = (uint32_t)M * 4u;
    const int b_nc = wave % NC;
    int b_ih0 = 0, b_iw0 = 0, b_base = 0;
    uint32_t b_cbad = 0;
    if constexpr (EPI != 2) {
        const int col = n0 + b_nc * 64 + lane;
        const int n = col / OHW;
        const int pix = col - n * OHW;
        const int i = pix / p.OW;
        const int j = pix - i * p.OW;
        b_ih0 = i * sh - p.ph;
        b_iw0 = j * sw - p.pw;
        b_base = (n * p.Cin + g * Cin_g) * IHW + b_ih0 * IW + b_iw0;
        b_cbad = col < p.Ncol ? 0u : kOob;
    }
    auto b_row = [&](int q) { return (wave + NW * q) / NC; };

    // Dense B (EPI 2): B[r][col] row-major with Ncol columns, the row offset
    // in the scalar offset.  Columns past Ncol, and rows past R (only when
    // R % TK != 0), get the out-of-range offset alone in the lane offset and
    // read 0.
    const uint32_t b_dvoff =
        n0 + b_nc * 64 + lane < p.Ncol ? (uint32_t)(n0 + b_nc * 64 + lane) * 4u : kOob;
    auto copy_b_dense = [&](BTile& dst, int kbase) {
#pragma unroll
        for (int q = 0; q < NB; ++q) {
            const int r = kbase + b_row(q);
            const bool rok = TAP || r < R;
            copy_to_lds(rx, &dst[b_row(q)][b_nc * 64], rok ? b_dvoff : kOob,
                        rok ? (uint32_t)r * (uint32_t)p.Ncol * 4u : 0u);
        }
    };

    auto copy_a = [&](ATile& dst, int kbase) {
#pragma unroll
        for (int q = 0; q < NA; ++q) {
            float* d = &dst[0][0] + 64 * (wave + NW * q);
            if constexpr (A_UNIFORM) {
                const int k = 64 * (wave + NW * q) / TM;
                const uint32_t mo = (uint32_t)(64 * (wave + NW * q) - k * TM) * 4u;
                // (the channel-blocked order covers R in whole stages, R % TK == 0)
                const bool rok = TAP || kbase + k < R;
                copy_to_lds(ra, d, rok ? a_voff[0] : kOob,
                            rok ? (uint32_t)(kbase + k) * a_row4 + mo : 0u);
            } else if constexpr (TAP) {
                copy_to_lds(ra, d, a_voff[q], (uint32_t)kbase * a_row4);
            } else if (kbase + TK <= R) {  // a whole stage: no row past R
                copy_to_lds(ra, d, a_voff[q], (uint32_t)kbase * a_row4);
            } else {
                // k varies across the wave: the scalar offset stays the
                // stage's (wave-uniform) and a row past R gets the
                // out-of-range offset alone, which the scalar offset cannot
                // carry back into range
                copy_to_lds(ra, d, kbase + a_k[q] < R ? a_voff[q] : kOob,
                            (uint32_t)kbase * a_row4);
            }
        }
    };

    // Channel-blocked order r = (c / TK, u, v, c % TK) (or tap-major
    // (u, v, c)): a stage covers TK channels of a single tap (u, v), so the
    // column's bounds test and address are formed once per stage and each
    // copy only adds its channel's plane offset as the uniform soffset.
    auto copy_b_tap = [&](BTile& dst, int u, int v, int c0) {
        const int ih = b_ih0 + u;
        const int iw = b_iw0 + v;
        // (a column past Ncol or a tap outside the image takes the
        // out-of-range offset alone: with the channel's scalar offset added
        // it stays out of range)
        const bool ok = b_cbad == 0u && (unsigned)ih < (unsigned)IH && (unsigned)iw < (unsigned)IW;
        const uint32_t voff = ok ? (uint32_t)(b_base + u * IW + v) * 4u : kOob;
#pragma unroll
        for (int q = 0; q < NB; ++q)
            copy_to_lds(rx, &dst[b_row(q)][b_nc * 64], voff,
                        (uint32_t)((c0 + b_row(q)) * IHW) * 4u);
    };

    // Channel-major order r = (c, u, v) for any Cin_g.  The tap decomposition
    // is wave-uniform (scalar).  Out-of-range taps get an offset with bit 31
    // set; a wave whose columns all have their whole window inside the image
    // (every wave of an unpadded layer) skips the per-tap bounds test.
    const bool b_inside =
        b_ih0 >= 0 && b_ih0 + kh <= IH && b_iw0 >= 0 && b_iw0 + kw <= IW;
    const bool b_all_inside = __all(b_inside);
    // A wave's copies of a stage take rows r0, r0 + STEP, r0 + 2 STEP, ...
    // (STEP = NW / NC): (c, u, v) and the plane offset of r0 come from one
    // division per stage, the later rows from a scalar walk (one tap at a
    // time, carrying v into u and u into c).
    constexpr int STEP = NW / NC;
    static_assert(STEP * NC == NW, "B copy rows advance by a whole step");
    // With a tap table and every window inside the image, a copy's tap
    // offset is a table entry, moved to the scalar offset with one lane
    // read: lane i < 16 of tap_v holds entry kbase + wave / NC + i of the
    // next stage to copy (the wave's rows are kbase + wave / NC + STEP*q).
    // Rows past R read the entry X_bytes: out of range.
    const bool use_taps = p.taps != nullptr && b_all_inside;
    const __amdgpu_buffer_rsrc_t rtap =
        make_rsrc(p.taps, p.taps ? (uint32_t)((R + TK - 1) / TK * TK) * 4u : 0u);
    const uint32_t b_voff4 = ((uint32_t)b_base * 4u) | b_cbad;
    uint32_t tap_v = 0;
    auto load_taps = [&](int kbase) {
        tap_v = __builtin_amdgcn_raw_buffer_load_b32(
            rtap, (uint32_t)(kbase + wave / NC + (lane & 15)) * 4u, 0, 0);
    };
    auto copy_b_any = [&](BTile& dst, int kbase) {
        if (use_taps) {
            // all lane reads first: a scalar offset read right after the
            // lane read that writes it costs wait states per copy
            uint32_t soff[NB];
#pragma unroll
            for (int q = 0; q < NB; ++q)
                soff[q] = (uint32_t)__builtin_amdgcn_readlane((int)tap_v, STEP * q);
#pragma unroll
            for (int q = 0; q < NB; ++q)
                copy_to_lds(rx, &dst[b_row(q)][b_nc * 64], b_voff4, soff[q]);
            return;
        }
        int r = kbase + b_row(0);
        int c = r / khw;
        int u = (r - c * khw) / kw;
        int v = r - c * khw - u * kw;
        int off = c * IHW + u * IW + v;
        // (carries as 0/1 arithmetic: straight-line scalar code, no branch
        // per row)
        auto advance = [&]() {
#pragma unroll
            for (int t = 0; t < STEP; ++t) {
                ++r;
                ++v;
                ++off;
                const int cv = v == kw;
                v -= cv * kw;
                u += cv;
                off += cv * (IW - kw);
                const int cu = u == kh;
                u -= cu * kh;
                off += cu * (IHW - kh * IW);
            }
        };
        if (b_all_inside) {  // no tap leaves the image: no per-tap test
#pragma unroll
            for (int q = 0; q < NB; ++q) {
                const uint32_t bad = (r < R ? 0u : kOob) | b_cbad;
                copy_to_lds(rx, &dst[b_row(q)][b_nc * 64], ((uint32_t)(b_base + off) * 4u) | bad,
                            0u);
                advance();
            }
        } else {
#pragma unroll
            for (int q = 0; q < NB; ++q) {
                const int ih = b_ih0 + u;
                const int iw = b_iw0 + v;
                const uint32_t bad = (r < R ? 0u : kOob) | b_cbad |
                                     (((uint32_t)((unsigned)ih >= (unsigned)IH) |
                                       (uint32_t)((unsigned)iw >= (unsigned)IW)) << 31);
                copy_to_lds(rx, &dst[b_row(q)][b_nc * 64], ((uint32_t)(b_base + off) * 4u) | bad,
                            0u);
                advance();
            }
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
            // (a tail split's partials leave the bias to the reduce)
            const __amdgpu_buffer_rsrc_t rbias =
                make_rsrc(p.bias, p.bias && !tail ? (uint32_t)(p.G * M) * 4u : 0u);
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

    const int nst_all = (R + TK - 1) / TK;
    const bool splitk = EPI >= 2 || tail;
    const int sps = EPI >= 2 ? p.stages_per_split : p.tail_sps;
    const int s_begin = splitk ? split * sps : 0;
    const int nst = splitk ? min(nst_all, s_begin + sps) : nst_all;
    // blocked walk state: stage s covers tap (tu, tv) of channels tc .. tc + TK - 1.
    // It is updated in the loop body itself: captured by reference in a
    // lambda, it was kept in scratch memory, and the scratch accesses' waits
    // also stalled on the next stage's global loads.
    int tu = 0, tv = 0, tc = 0;
    if constexpr (EPI != 2 && TAP) {
        // the walk state of the split's first stage
        if (p.blocked) {  // stage s: channels (s / khw) * TK.., tap s % khw
            const int t = s_begin % khw;
            tc = (s_begin / khw) * TK;
            tu = t / kw;
            tv = t - tu * kw;
        } else {          // stage s: channels (s * TK) % Cin_g.., tap (s * TK) / Cin_g
            const int t = (s_begin * TK) / Cin_g;
            tc = s_begin * TK - t * Cin_g;
            tu = t / kw;
            tv = t - tu * kw;
        }
    }

    copy_a(As0, s_begin * TK);
    if constexpr (EPI == 2) {
        copy_b_dense(Bs0, s_begin * TK);
    } else if constexpr (TAP) {
        copy_b_tap(Bs0, tu, tv, tc);
    } else {
        if (use_taps)
            load_taps(s_begin * TK);
        copy_b_any(Bs0, s_begin * TK);
        if (use_taps)
            load_taps((s_begin + 1) * TK);
    }
    __builtin_amdgcn_s_waitcnt(kVmcnt0);
    __syncthreads();

    const int arow = wm * MI * MT + lane % MT;
    const int bcol = wn * NI * MT + lane % MT;
    const int kl = lane / MT;

    // The stage loop is unrolled by two so that each half has its buffers
    // fixed: half h copies stage s + h + 1 into buffer 1 - h and multiplies
    // the fragments of stage s + h from buffer h.
    for (int s0 = s_begin; s0 < nst; s0 += 2) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int s = s0 + h;
            if (s >= nst)
                break;
            ATile& Ac = h ? As1 : As0;
            BTile& Bc = h ? Bs1 : Bs0;
            ATile& An = h ? As0 : As1;
            BTile& Bn = h ? Bs0 : Bs1;
            if (s + 1 < nst) {
                copy_a(An, (s + 1) * TK);
                if constexpr (EPI == 2) {
                    copy_b_dense(Bn, (s + 1) * TK);
                } else if constexpr (TAP) {
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
                    copy_b_tap(Bn, tu, tv, tc);
                } else {
                    copy_b_any(Bn, (s + 1) * TK);
                    if (use_taps)  // (past the end it reads 0, unused)
                        load_taps((s + 2) * TK);
                }
            }
            __builtin_amdgcn_sched_barrier(0);
            // Rolling fragment prefetch: the LDS reads of k-step ks + PF are
            // issued before the MFMAs of k-step ks (a ring of PF + 1 fragment
            // sets).  The scheduling barriers pin that order; left alone, the
            // scheduler trades it for fewer registers and waits on LDS before
            // every k-step.
            constexpr int PF = KS > 2 ? 2 : KS - 1;
            float fa[PF + 1][MI], fb[PF + 1][NI];
#pragma unroll
            for (int ks = 0; ks < KS + PF; ++ks) {
                if (ks < KS) {  // fragments of k-step ks into ring slot ks % (PF + 1)
#pragma unroll
                    for (int mi = 0; mi < MI; ++mi)
                        fa[ks % (PF + 1)][mi] = Ac[ks * Op::kStep + kl][arow + mi * MT];
#pragma unroll
                    for (int ni = 0; ni < NI; ++ni)
                        fb[ks % (PF + 1)][ni] = Bc[ks * Op::kStep + kl][bcol + ni * MT];
                }
                if (ks >= PF) {  // MFMAs of k-step ks - PF
                    const int k = ks - PF;
                    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
                        for (int ni = 0; ni < NI; ++ni)
                            acc[mi][ni] = Op::run(fa[k % (PF + 1)][mi], fb[k % (PF + 1)][ni],
                                                  acc[mi][ni]);
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
            // the next stage's copies have landed in LDS, for every wave
            __builtin_amdgcn_s_waitcnt(kVmcnt0);
            __syncthreads();
        }
    }

    // ---- epilogue (branch-free: masked lanes store to an out-of-range offset)
    const __amdgpu_buffer_rsrc_t ry = make_rsrc(p.Y, p.Y_bytes);
    // Masks are folded into the offsets with integer ops (bit 31 = past the
    // buffer, dropped by the hardware): short-circuit tests here become
    // divergent branches and make the compiler copy every accumulator out of
    // the AGPRs at once.
    // the wave's 64 columns, one per lane, rows regrouped by WaveRows
    typedef WaveRows<MT> WR;
    static_assert(NI * MT == 64, "a wave covers 64 columns");
    constexpr int NR = WR::kRows;
    const int wcol = n0 + wn * NI * MT + lane;
    if constexpr (EPI < 2) {
        if (tail) {
            // tail-split partial Pt[split][m][col - tail_c0] (the last group's)
            const __amdgpu_buffer_rsrc_t rp = make_rsrc(p.Pt, p.Pt_bytes);
            const int Nc = p.Ncol - p.tail_c0;
            const uint32_t cbad = (uint32_t)(wcol >= p.Ncol) << 31;
#pragma unroll
            for (int mi = 0; mi < MI; ++mi) {
#pragma unroll
                for (int q = 0; q < Op::kRegs; ++q) {
                    float v[NR];
                    wave_rows<MT>(acc[mi], q, v);
#pragma unroll
                    for (int h = 0; h < NR; ++h) {
                        const int m = m0 + wm * MI * MT + mi * MT + WR::row(q, h);
                        const uint32_t off =
                            ((uint32_t)((split * M + m) * Nc + wcol - p.tail_c0) * 4u) | cbad |
                            ((uint32_t)(m >= M) << 31);
                        buf_st_f32(v[h], rp, off);
                    }
                }
            }
            return;
        }
    }
    if constexpr (EPI >= 2) {
        // split partial P[split][g][m][col], lanes along col
        const uint32_t cbad = (uint32_t)(wcol >= p.Ncol) << 31;
#pragma unroll
        for (int mi = 0; mi < MI; ++mi) {
#pragma unroll
            for (int q = 0; q < Op::kRegs; ++q) {
                float v[NR];
                wave_rows<MT>(acc[mi], q, v);
#pragma unroll
                for (int h = 0; h < NR; ++h) {
                    const int m = m0 + wm * MI * MT + mi * MT + WR::row(q, h);
                    const uint32_t off =
                        ((uint32_t)(((split * p.G + g) * M + m) * p.Ncol + wcol) * 4u) | cbad |
                        ((uint32_t)(m >= M) << 31);
                    buf_st_f32(v[h], ry, off);
                }
            }
        }
    } else if constexpr (EPI == 0) {
        const int n = wcol / OHW;
        const int pix = wcol - n * OHW;
        const int cbase = n * p.Cout * OHW + pix;
        const uint32_t cbad = (uint32_t)(wcol >= p.Ncol) << 31;
#pragma unroll
        for (int mi = 0; mi < MI; ++mi) {
#pragma unroll
            for (int q = 0; q < Op::kRegs; ++q) {
                float z[NR];
                wave_rows<MT>(acc[mi], q, z);
#pragma unroll
                for (int h = 0; h < NR; ++h) {
                    const int m = m0 + wm * MI * MT + mi * MT + WR::row(q, h);
                    const int oc = g * M + m;
                    // ReLU: non-positive values (NaN included) become 0; without
                    // ReLU every value passes unchanged
                    const float v = z[h] > 0.f ? z[h] : (p.relu ? 0.f : z[h]);
                    const uint32_t off = ((uint32_t)(cbase + oc * OHW) * 4u) | cbad |
                                         ((uint32_t)(m >= M) << 31);
                    buf_st_f32(v, ry, off);
                }
            }
        }
    } else {
        const int pss = p.psh * p.psw;
        const int OutHW = p.OutH * p.OutW;
        const __amdgpu_buffer_rsrc_t rom = make_rsrc(MASK ? p.Omask : p.Y, p.Y_bytes);
        const bool cok = wcol < p.Ncol;
        const int n = cok ? wcol / OHW : 0;
        const int pix = wcol - n * OHW;
        const int a = pix / p.OW;
        const int b = pix - a * p.OW;
        const int hb = cok ? p.psh * (a + p.a0h) - p.oph : -(1 << 28);
        const int wb = p.psw * (b + p.a0w) - p.opw;
        const int cb = (n * p.Cout + g * p.Cg_out) * OutHW;
        // per MT-row block: every position (and, masked, every value of the
        // ReLU output) first, then the stores (a load after a store to
        // another buffer could not be moved above it, so each would wait
        // alone).  Masked, a 32-row block goes in two halves of its
        // registers: the mask values and offsets of a whole block beside the
        // accumulators took the kernel past 128 VGPRs (three waves per SIMD
        // instead of four).
        constexpr int QC = MASK && Op::kRegs > 8 ? Op::kRegs / 2 : Op::kRegs;
#pragma unroll
        for (int mi = 0; mi < MI; ++mi) {
#pragma unroll
          for (int q0 = 0; q0 < Op::kRegs; q0 += QC) {
            uint32_t off[QC][NR];
            float y[QC][NR];
#pragma unroll
            for (int qq = 0; qq < QC; ++qq) {
                const int q = q0 + qq;
#pragma unroll
                for (int h = 0; h < NR; ++h) {
                    const int m = m0 + wm * MI * MT + mi * MT + WR::row(q, h);
                    int c = m, fh = 0, fw = 0;
                    if (pss != 1) {
                        c = (int)fdiv((uint32_t)m, p.div_pss);
                        const int fr = m - c * pss;
                        fh = (int)fdiv((uint32_t)fr, p.div_psw);
                        fw = fr - fh * p.psw;
                    }
                    const int hh = hb + fh;
                    const int ww = wb + fw;
                    const uint32_t bad = ((uint32_t)(m >= M) |
                                          (uint32_t)((unsigned)hh >= (unsigned)p.OutH) |
                                          (uint32_t)((unsigned)ww >= (unsigned)p.OutW))
                                         << 31;
                    off[qq][h] = ((uint32_t)(cb + c * OutHW + hh * p.OutW + ww) * 4u) | bad;
                    // backward of the ReLU that produced the gather target:
                    // keep the gradient only where that output was > 0
                    if constexpr (MASK)
                        y[qq][h] = buf_ld_f32(rom, off[qq][h]);
                }
            }
#pragma unroll
            for (int qq = 0; qq < QC; ++qq) {
                float v[NR];
                wave_rows<MT>(acc[mi], q0 + qq, v);
#pragma unroll
                for (int h = 0; h < NR; ++h) {
                    if constexpr (MASK)
                        v[h] = y[qq][h] > 0.f ? v[h] : 0.f;
                    buf_st_f32(v[h], ry, off[qq][h]);
                }
            }
          }
        }
    }
}

// Forward weights, transposed for the LDS copies and reordered to the
// reduction order: Wp[g][r][m] = W[g*M + m][c][t] (t = u*kw + v) with
//   order > 0:  r = ((c / tk) * khw + t) * tk + c % tk    (channel-blocked)
//   order < 0:  r = t * Cg + c                             (tap-major)
//   order == 0: r = c * khw + t                            (channel-major)
__global__ void __launch_bounds__(256)
pack_weights_kernel(const float* __restrict__ W, float* __restrict__ Wp, int G, int M, int Cg,
                    int khw, int tk, int order)
{
    const int R = Cg * khw;
    const long total = (long)G * M * R;
    for (long e = blockIdx.x * (long)blockDim.x + threadIdx.x; e < total;
         e += (long)gridDim.x * blockDim.x) {
        const int m = (int)(e % M);
        const long gr = e / M;
        const int r = (int)(gr % R);
        const int g = (int)(gr / R);
        int c, t;
        if (order > 0) {
            const int ci = r % tk;
            t = (r / tk) % khw;
            c = (r / (tk * khw)) * tk + ci;
        } else if (order < 0) {
            t = r / Cg;
            c = r - t * Cg;
        } else {
            c = r / khw;
            t = r - c * khw;
        }
        Wp[e] = W[((long)(g * M + m) * Cg + c) * khw + t];
    }
}

hipError_t launch_pack_weights(const float* W, float* Wp, int G, int M, int Cg, int khw, int tk,
                               int order, hipStream_t s)
{
    const long total = (long)G * M * Cg * khw;
    if (total == 0)
        return hipSuccess;
    long blocks = (total + 255) / 256;
    if (blocks > 4096)
        blocks = 4096;
    hipLaunchKernelGGL(pack_weights_kernel, dim3((unsigned)blocks), dim3(256), 0, s, W, Wp, G, M,
                       Cg, khw, tk, order);
    return hipGetLastError();
}

__global__ void __launch_bounds__(256)
tap_table_kernel(uint32_t* __restrict__ T, int rpad, int R, int kh, int kw, int IHW, int IW,
                 uint32_t oob)
{
    const int r = blockIdx.x * 256 + threadIdx.x;
    if (r >= rpad)
        return;
    uint32_t e = oob;
    if (r < R) {
        const int khw = kh * kw;
        const int c = r / khw;
        const int t = r - c * khw;
        const int u = t / kw;
        e = (uint32_t)(c * IHW + u * IW + (t - u * kw)) * 4u;
    }
    T[r] = e;
}

hipError_t launch_tap_table(uint32_t* T, int rpad, int R, int kh, int kw, int IHW, int IW,
                            uint32_t oob, hipStream_t s)
{
    if (rpad <= 0)
        return hipSuccess;
    hipLaunchKernelGGL(tap_table_kernel, dim3((unsigned)((rpad + 255) / 256)), dim3(256), 0, s, T,
                       rpad, R, kh, kw, IHW, IW, oob);
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
    int64_t tiles = (int64_t)((p.Ncol + TN - 1) / TN) * ((p.M + TM - 1) / TM) * p.G;
    int64_t per_xcd;  // 8 XCDs; see the kernel's tile order
    if (EPI < 2 && p.tail_splits > 1) {
        const int64_t items = (tiles - p.tail_T) * p.tail_splits;
        per_xcd = (p.tail_T + 7) / 8 + (items + 7) / 8;
    } else {
        if (EPI >= 2)
            tiles *= p.splits;
        per_xcd = (tiles + 7) / 8;
    }
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
    if ((EPI == 0 || EPI == 3) && p.kh == 11 && p.kw == 11 && p.sh == 4 && p.sw == 4)
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

namespace {
template <int MT, int WM, int WN, int MI, int NI, int TK>
hipError_t launch_dense(const ConvGemmParams& p, hipStream_t s)
{
    // whole stages (R % TK == 0) need no masking of the reduction tail
    if (p.R % TK == 0)
        return launch_one<MT, WM, WN, MI, NI, TK, 0, 0, 0, 0, 2, true, false>(p, s);
    return launch_one<MT, WM, WN, MI, NI, TK, 0, 0, 0, 0, 2, false, false>(p, s);
}
}  // namespace

hipError_t launch_dense_gemm_f32(const ConvGemmParams& p, int tile, hipStream_t s)
{
    if (p.Ncol == 0 || p.M == 0)
        return hipSuccess;
    if (p.G != 1 || p.splits < 1 || p.stages_per_split < 1)
        return hipErrorInvalidValue;
    switch (tile) {
    case TILE_128x128:
        return launch_dense<32, 2, 2, 2, 2, 16>(p, s);
    case TILE_96x256:
        return launch_dense<32, 1, 4, 3, 2, 16>(p, s);
    case TILE_48x256:
        return launch_dense<16, 1, 4, 3, 4, 16>(p, s);
    case TILE_64x256:
        return launch_dense<32, 1, 4, 2, 2, 16>(p, s);
    default:
        return hipErrorInvalidValue;
    }
}

// ---------------------------------------------------------------------------
// Dense split-K GEMM with both operands reduction-contiguous:
// P[split][m][n] = sum over the split's range of r of A[m][r] B[n][r]
// (A = p.A, M x R; B = p.X, Ncol x R; P = p.Y).  The inner-product forward
// pass (Y[n][k] = sum_c X[n][c] W[k][c]) reads its operands as stored.
//
// A stage is 16 deep: each operand row contributes 16 consecutive floats,
// four 16-byte chunks, copied global -> LDS by 16-byte DMA (a wave copy =
// 16 rows).  In LDS, logical chunk c of row r sits in slot c ^ kc_swz(r);
// the fragment reads (ds_read_b128 of one chunk of 16 consecutive rows) then
// touch distinct banks.  The MFMA k index is permuted within a stage: lane
// group q (lane / MT) takes the stage's k = q * (16 / (64 / MT)) + step, so a
// lane's values for the whole stage are consecutive floats of one row.  A and
// B use the same permutation, so the sum over the stage is unchanged.
__device__ __forceinline__ int kc_swz(int r)
{
    return ((r >> 2) & 1) | ((((r >> 1) ^ (r >> 3)) & 1) << 1);
}

__device__ __forceinline__ void copy16_to_lds(__amdgpu_buffer_rsrc_t r, float* dst, uint32_t voff,
                                              uint32_t soff)
{
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)dst, 16, voff, soff, 0, 0);
}

template <int MT, int WM, int WN, int MI, int NI, bool FULL>
__global__ void __launch_bounds__(64 * WM * WN)
dense_gemm_nt_kernel(const ConvGemmParams p)
{
    typedef Mfma<MT> Op;
    constexpr int TK = 16;
    constexpr int NW = WM * WN;
    constexpr int TM = WM * MI * MT;
    constexpr int TN = WN * NI * MT;
    constexpr int CA = TM / 16, CB = TN / 16;  // 16-row wave copies per stage
    constexpr int NA = (CA + NW - 1) / NW, NB = (CB + NW - 1) / NW;
    constexpr int KL = TK / (64 / MT);        // stage k values per lane: 8 or 4
    constexpr int NCH = KL / 4;               // 16-byte chunks per lane and row
    static_assert(TK / Op::kStep == KL, "one k value per lane per MFMA step");
    __shared__ floatx4 As0[TM * 4], As1[TM * 4], Bs0[TN * 4], Bs1[TN * 4];
    typedef floatx4 ATile[TM * 4];
    typedef floatx4 BTile[TN * 4];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave % WM;
    const int wn = wave / WM;
    // XCD-contiguous tile order, row tiles fastest, the split slowest
    const int n_mt = (p.M + TM - 1) / TM;
    const int n_ct = (p.Ncol + TN - 1) / TN;
    const int per_xcd = gridDim.x >> 3;
    const int T = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
    if (T >= n_mt * n_ct * p.splits)
        return;
    const int mt = T % n_mt;
    const int ct = (T / n_mt) % n_ct;
    const int split = T / (n_mt * n_ct);
    const int m0 = mt * TM, n0 = ct * TN;
    const int M = p.M, R = p.R;

    const __amdgpu_buffer_rsrc_t ra = make_rsrc(p.A, p.A_bytes);
    const __amdgpu_buffer_rsrc_t rb = make_rsrc(p.X, p.X_bytes);

    // copy lane mapping: row lane / 4 of the copy's 16, logical chunk
    // (lane % 4) ^ kc_swz(row) -> LDS slot lane % 4 of that row
    const int crow = lane >> 2;
    const int cch = (lane & 3) ^ kc_swz(crow);
    uint32_t a_off[NA], b_off[NB];
#pragma unroll
    for (int q = 0; q < NA; ++q) {
        const int row = m0 + (wave + NW * q) * 16 + crow;
        a_off[q] = row < M ? (uint32_t)(row * R + 4 * cch) * 4u : kOob;
    }
#pragma unroll
    for (int q = 0; q < NB; ++q) {
        const int col = n0 + (wave + NW * q) * 16 + crow;
        b_off[q] = col < p.Ncol ? (uint32_t)(col * R + 4 * cch) * 4u : kOob;
    }
    // stage k base in the scalar offset; past the reduction's end (R % 16 != 0)
    // a chunk reads 0 (R % 4 == 0: a chunk never straddles the end)
    auto tail = [&](uint32_t off, int kbase) -> uint32_t {
        if constexpr (FULL)
            return off;
        else
            return kbase + 4 * cch < R ? off : kOob;
    };
    auto copy_stage = [&](ATile& a, BTile& b, int kbase) {
#pragma unroll
        for (int q = 0; q < NA; ++q)
            if (CA % NW == 0 || wave + NW * q < CA)
                copy16_to_lds(ra, (float*)&a[(wave + NW * q) * 64], tail(a_off[q], kbase),
                              (uint32_t)kbase * 4u);
#pragma unroll
        for (int q = 0; q < NB; ++q)
            if (CB % NW == 0 || wave + NW * q < CB)
                copy16_to_lds(rb, (float*)&b[(wave + NW * q) * 64], tail(b_off[q], kbase),
                              (uint32_t)kbase * 4u);
    };

    typename Op::acc_t acc[MI][NI];
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int ni = 0; ni < NI; ++ni)
            acc[mi][ni] = typename Op::acc_t{};

    const int nst_all = (R + TK - 1) / TK;
    const int s_begin = split * p.stages_per_split;
    const int nst = min(nst_all, s_begin + p.stages_per_split);
    copy_stage(As0, Bs0, s_begin * TK);
    __builtin_amdgcn_s_waitcnt(kVmcnt0);
    __syncthreads();

    // fragment slots: row i = lane % MT of each MT-row block, logical chunks
    // (lane / MT) * NCH + t
    const int fi = lane % MT;
    const int fq = lane / MT;
    int fslot[NCH];
#pragma unroll
    for (int t = 0; t < NCH; ++t)
        fslot[t] = fi * 4 + ((fq * NCH + t) ^ kc_swz(fi & 15));
    const int arow0 = wm * MI * MT, bcol0 = wn * NI * MT;

    for (int s0 = s_begin; s0 < nst; s0 += 2) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int s = s0 + h;
            if (s >= nst)
                break;
            ATile& Ac = h ? As1 : As0;
            BTile& Bc = h ? Bs1 : Bs0;
            ATile& An = h ? As0 : As1;
            BTile& Bn = h ? Bs0 : Bs1;
            if (s + 1 < nst)
                copy_stage(An, Bn, (s + 1) * TK);
            __builtin_amdgcn_sched_barrier(0);
            floatx4 fa[NCH][MI], fb[NCH][NI];
#pragma unroll
            for (int t = 0; t < NCH; ++t) {
#pragma unroll
                for (int mi = 0; mi < MI; ++mi)
                    fa[t][mi] = Ac[(arow0 + mi * MT) * 4 + fslot[t]];
#pragma unroll
                for (int ni = 0; ni < NI; ++ni)
                    fb[t][ni] = Bc[(bcol0 + ni * MT) * 4 + fslot[t]];
            }
#pragma unroll
            for (int t = 0; t < NCH; ++t)
#pragma unroll
                for (int u = 0; u < 4; ++u)
#pragma unroll
                    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
                        for (int ni = 0; ni < NI; ++ni)
                            acc[mi][ni] = Op::run(fa[t][mi][u], fb[t][ni][u], acc[mi][ni]);
            __builtin_amdgcn_s_waitcnt(kVmcnt0);
            __syncthreads();
        }
    }

    // split partial P[split][m][col]: the wave's 64 columns, one per lane,
    // rows regrouped by WaveRows
    const __amdgpu_buffer_rsrc_t ry = make_rsrc(p.Y, p.Y_bytes);
    typedef WaveRows<MT> WR;
    static_assert(NI * MT == 64, "a wave covers 64 columns");
    constexpr int NR = WR::kRows;
    const int col = n0 + bcol0 + lane;
    const uint32_t cbad = (uint32_t)(col >= p.Ncol) << 31;
#pragma unroll
    for (int mi = 0; mi < MI; ++mi) {
#pragma unroll
        for (int q = 0; q < Op::kRegs; ++q) {
            float v[NR];
            wave_rows<MT>(acc[mi], q, v);
#pragma unroll
            for (int h = 0; h < NR; ++h) {
                const int m = m0 + arow0 + mi * MT + WR::row(q, h);
                const uint32_t off = ((uint32_t)((split * M + m) * p.Ncol + col) * 4u) | cbad |
                                     ((uint32_t)(m >= M) << 31);
                buf_st_f32(v[h], ry, off);
            }
        }
    }
}

namespace {
template <int MT, int WM, int WN, int MI, int NI>
hipError_t launch_nt(const ConvGemmParams& p, hipStream_t s)
{
    constexpr int TM = WM * MI * MT, TN = WN * NI * MT;
    const int64_t tiles =
        (int64_t)((p.Ncol + TN - 1) / TN) * ((p.M + TM - 1) / TM) * p.splits;
    const int64_t per_xcd = (tiles + 7) / 8;
    if (p.R % 16 == 0)
        hipLaunchKernelGGL((dense_gemm_nt_kernel<MT, WM, WN, MI, NI, true>),
                           dim3((unsigned)(per_xcd * 8)), dim3(64 * WM * WN), 0, s, p);
    else
        hipLaunchKernelGGL((dense_gemm_nt_kernel<MT, WM, WN, MI, NI, false>),
                           dim3((unsigned)(per_xcd * 8)), dim3(64 * WM * WN), 0, s, p);
    return hipGetLastError();
}
}  // namespace

// Compute units of the current device (queried once; 256 when no device
// answers).
int device_cu_count()
{
    static int cus = 0;
    if (cus > 0)
        return cus;
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        n <= 0) {
        (void)hipGetLastError();
        return 256;
    }
    cus = n;
    return cus;
}

hipError_t launch_dense_gemm_nt_f32(const ConvGemmParams& p, int tile, hipStream_t s)
{
    if (p.Ncol == 0 || p.M == 0)
        return hipSuccess;
    if (p.R % 4 != 0 || p.splits < 1 || p.stages_per_split < 1 ||
        (((uintptr_t)p.A | (uintptr_t)p.X) & 15) != 0)
        return hipErrorInvalidValue;
    switch (tile) {
    case TILE_128x128:
        return launch_nt<32, 2, 2, 2, 2>(p, s);
    case TILE_96x256:
        return launch_nt<32, 1, 4, 3, 2>(p, s);
    case TILE_48x256:
        return launch_nt<16, 1, 4, 3, 4>(p, s);
    case TILE_64x256:
        return launch_nt<32, 1, 4, 2, 2>(p, s);
    default:
        return hipErrorInvalidValue;
    }
}

hipError_t launch_conv_gemm_f32(const ConvGemmParams& p, int epi, int tile, bool tap_major,
                                hipStream_t s)
{
    if (p.Ncol == 0)
        return hipSuccess;
    if (tile < 0 || tile >= TILE_COUNT || (tap_major && p.Cin_g % kTiles[tile].tk != 0))
        return hipErrorInvalidValue;
    if ((epi == 0 || epi == 1) && p.tail_splits > 1) {
        // the tail: whole column tiles of the last group, each range non-empty
        const TileShape& t = kTiles[tile];
        const int tm = t.wm * t.mi * t.mt, tn = t.wn * t.ni * t.mt;
        const int n_mt = (p.M + tm - 1) / tm, n_ct = (p.Ncol + tn - 1) / tn;
        const int n_tiles = n_mt * n_ct * p.G;
        const int nst = (p.R + t.tk - 1) / t.tk;
        if (p.tail_T < (p.G - 1) * n_mt * n_ct || p.tail_T >= n_tiles || p.tail_T % n_mt != 0 ||
            p.tail_c0 != (p.tail_T / n_mt) % n_ct * tn || p.tail_sps < 1 ||
            (int64_t)(p.tail_splits - 1) * p.tail_sps >= nst ||
            (int64_t)p.tail_splits * p.M * (p.Ncol - p.tail_c0) * 4 > (int64_t)p.Pt_bytes ||
            p.Pt == nullptr)
            return hipErrorInvalidValue;
    }
    if (epi == 0)
        return launch_tile<0, false>(p, tile, tap_major, s);
    if (epi == 3) {
        if (p.splits < 1 || p.stages_per_split < 1)
            return hipErrorInvalidValue;
        return launch_tile<3, false>(p, tile, tap_major, s);
    }
    return p.Omask ? launch_tile<1, true>(p, tile, tap_major, s)
                   : launch_tile<1, false>(p, tile, tap_major, s);
}

}  // namespace caffe_hip
