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
// Both operands are copied global -> LDS by 16-byte DMA in 64-deep stages:
// each operand row contributes 8 chunks of 8 bf16 (128 bytes, one cache line
// when aligned) per stage.  One wave copy moves 8 rows: lane l takes row
// l / 8 and lands at slot l % 8 of that row's 128 bytes, the row's chunks
// in order along the lanes (the address unit then handles whole lines; a
// copy whose lanes step across rows runs at a quarter of the rate).  Inside
// a row, chunk c sits at slot c ^ chunk_swz(row), so that the fragment reads
// (one chunk of consecutive rows across the lanes) hit distinct banks
// whether the LDS serves 8 or 16 lanes of 16 bytes per cycle.
//
// A rows are contiguous in global memory.  A B row is one output column:
// its chunk kc = (u, vg, c8) sits at a byte offset from the column's pixel
// that does not depend on the column (see GemmBf16Params), so each lane
// walks its one chunk index per stage and adds the offset to the pixel base
// of each of its columns.  Past the last
// chunk the offset is out of range (the copy lands zeros).  Columns past
// Ncol re-read the last column; their results are never stored.
__device__ __forceinline__ void copy16_lds(__amdgpu_buffer_rsrc_t r, u32x4* dst, uint32_t voff,
                                           uint32_t soff)
{
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)dst, 16, voff, soff, 0, 0);
}

// Slot permutation of the 8 chunks of tile row r (bits 0..3 of r only).
__device__ __forceinline__ int chunk_swz(int r)
{
    return (r & 6) | ((r ^ (r >> 3)) & 1);
}

// Workgroup barrier between pipeline stages.  Each wave has already waited
// (vmcnt) for its own copies of the stage it is about to read, and its reads
// of the buffer the next copies overwrite were consumed by MFMAs before it
// arrives; __syncthreads would in addition wait for every copy still in
// flight (its release fence covers LDS DMA), serialising a deeper pipeline.
// The empty asm statements keep the compiler from moving LDS accesses across.
__device__ __forceinline__ void stage_barrier()
{
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// s_waitcnt vmcnt(n), expcnt and lgkmcnt left at their maxima.
template <int N>
__device__ __forceinline__ void wait_vmcnt()
{
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt(0x0F70 | (N & 15) | (((N >> 4) & 3) << 14));
}

// Workgroups of the bf16 GEMM that fit one compute unit's LDS at once: the
// register budget follows (one workgroup of 4 waves = one wave per SIMD may
// use the whole register file).
constexpr int bf16_gemm_blocks_per_cu(int tm, int tn, int ns)
{
    return (160 * 1024) / ((tm + tn) * kBf16TK * 2 * ns);
}

template <int MT, int WM, int WN, int MI, int NI, int NS, int EPI, int MASK>
__global__ void __launch_bounds__(64 * WM * WN,
                                  bf16_gemm_blocks_per_cu(WM * MI * MT, WN * NI * MT, NS))
conv_gemm_bf16_kernel(const GemmBf16Params p)
{
    typedef MfmaBf16<MT> Op;
    constexpr int NW = WM * WN;
    constexpr int TM = WM * MI * MT;
    constexpr int TN = WN * NI * MT;
    constexpr int TK = kBf16TK;       // reduction depth of a stage
    constexpr int CH = TK / 8;        // chunks per row per stage
    constexpr int RPI = 64 / CH;      // rows per wave copy
    constexpr int IA = TM / RPI;      // A copies per stage
    constexpr int NA = (IA + NW - 1) / NW;
    constexpr int NB = TN / RPI / NW; // B copies per wave per stage
    constexpr int KL = 64 / MT;       // lane groups along k of one instruction
    constexpr int KS = TK / Op::kK;   // instructions along k per stage
    static_assert(CH == 8 && NW % 2 == 0, "copy mapping: 8-chunk rows, swizzle by wave parity");
    static_assert(TM % RPI == 0 && TN % (RPI * NW) == 0 && MT % 16 == 0, "copy mapping");
    static_assert(Op::kK == 8 * KL && TK % Op::kK == 0, "stage depth");
    static_assert(NS == 2 || NS == 3, "buffers");

    __shared__ u32x4 A0[TM * CH], A1[TM * CH], A2[NS > 2 ? TM * CH : 1];
    __shared__ u32x4 B0[TN * CH], B1[TN * CH], B2[NS > 2 ? TN * CH : 1];

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
    const int M = p.M;
    const int OHW = p.OH * p.OW;

    const __amdgpu_buffer_rsrc_t ra = make_rsrc(p.A, p.A_bytes);
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(p.X, p.X_bytes);

    // copy i (= wave + NW*q) moves tile rows 8i .. 8i + 7; bit 3 of the row,
    // the only one of i in chunk_swz, is the wave's parity
    const int cr = lane >> 3;
    const int ck = (lane & 7) ^ chunk_swz(8 * wave + cr);  // this lane's chunk
    uint32_t a_voff[NA];
#pragma unroll
    for (int q = 0; q < NA; ++q) {
        const int row = m0 + RPI * (wave + NW * q) + cr;
        a_voff[q] = row < M ? ((uint32_t)((g * M + row) * p.Rp) + 8u * ck) * 2u : kOob;
    }
    uint32_t b_pix[NB];
#pragma unroll
    for (int q = 0; q < NB; ++q) {
        const int col = min(n0 + RPI * (wave + NW * q) + cr, p.Ncol - 1);
        const int n = (int)fdiv((uint32_t)col, p.div_ohw);
        const int pix = col - n * OHW;
        const int i = (int)fdiv((uint32_t)pix, p.div_ow);
        const int j = pix - i * p.OW;
        b_pix[q] = (uint32_t)(((n * p.IHp + i * p.sh + p.oh0) * p.IWp + j * p.sw + p.ow0) *
                                  p.Ctot + g * p.Cgp) * 2u;
    }
    // byte offset of this lane's chunk of stage t from a column's pixel
    auto b_delta = [&](int t) -> uint32_t {
        const int kc = t * CH + ck;
        if (p.blocked) {
            // stage t: 64-channel block t / ntap of tap t % ntap
            const int cb = (int)fdiv((uint32_t)t, p.div_ntap);
            const int tap = t - cb * p.ntap;
            const int u = (int)fdiv((uint32_t)tap, p.div_kw);
            const int vg = tap - u * p.kw;
            const uint32_t d =
                (uint32_t)(u * p.IWp * p.Ctot + vg * p.vstr + 8 * (cb * CH + ck)) * 2u;
            return kc < p.KC ? d : kOob;
        }
        const int tg = (int)fdiv((uint32_t)kc, p.div_cg8);
        const int c8 = kc - tg * p.Cg8;
        const int u = (int)fdiv((uint32_t)tg, p.div_kw);
        const int vg = tg - u * p.kw;
        const uint32_t d = (uint32_t)(u * p.IWp * p.Ctot + vg * p.vstr + 8 * c8) * 2u;
        return kc < p.KC ? d : kOob;
    };
    // The copies of one stage, NA + NB per wave, go out in KS parts, one
    // after each step of MFMAs: issued all at once they back up in the
    // address unit and stall the wave before its first MFMA.
    constexpr int NC = NA + NB;
    constexpr int CPP = (NC + KS - 1) / KS;  // copies per part
    auto issue_part = [&](int t, u32x4* As, u32x4* Bs, int part, uint32_t d) {
        const uint32_t soff = (uint32_t)(t * TK) * 2u;
#pragma unroll
        for (int c = part * CPP; c < (part + 1) * CPP && c < NC; ++c) {
            if (c < NA) {
                if (IA % NW == 0 || wave + NW * c < IA)
                    copy16_lds(ra, &As[(wave + NW * c) * 64], a_voff[c], soff);
            } else {
                copy16_lds(rx, &Bs[(wave + NW * (c - NA)) * 64], b_pix[c - NA] + d, 0u);
            }
        }
    };
    auto issue = [&](int t, u32x4* As, u32x4* Bs) {
        const uint32_t d = b_delta(t);
#pragma unroll
        for (int part = 0; part < KS; ++part)
            issue_part(t, As, Bs, part, d);
    };
    // this wave's copies of one stage (the vmcnt still allowed while the
    // next stage's copies are in flight)
    auto wait_all_but_next = [&]() {
        if constexpr (IA % NW == 0) {
            wait_vmcnt<NA + NB>();
        } else {
            if (wave < IA % NW)
                wait_vmcnt<NA + NB>();
            else
                wait_vmcnt<NA - 1 + NB>();
        }
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

    // fragment slots: tile row R = base + mi*MT + lane % MT, chunk
    // c = ks*KL + lane / MT at slot (R / 8)*64 + (R % 8)*8 + (c ^ chunk_swz(R));
    // chunk_swz(R) and (R % 8) do not change with mi (MT % 16 == 0) and
    // ks*KL only sets bits above lane / MT
    int fa[KS], fb[KS];
    {
        const int ra0 = wm * MI * MT + lane % MT;
        const int rb0 = wn * NI * MT + lane % MT;
        const int ea = (lane / MT) ^ chunk_swz(ra0);
        const int eb = (lane / MT) ^ chunk_swz(rb0);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            fa[ks] = (ra0 >> 3) * 64 + (ra0 & 7) * 8 + (ea ^ (ks * KL));
            fb[ks] = (rb0 >> 3) * 64 + (rb0 & 7) * 8 + (eb ^ (ks * KL));
        }
    }
    constexpr int FSTR = (MT / 8) * 64;  // next MT-row block

    // fragments of step ks + 1 are read while the instructions of step ks
    // run; after(ks) follows the instructions of step ks
    auto compute = [&](const u32x4* As, const u32x4* Bs, auto&& after) {
        bf16x8 xa[2][MI], xb[2][NI];
        auto read = [&](int ks, int b) {
#pragma unroll
            for (int mi = 0; mi < MI; ++mi)
                xa[b][mi] = __builtin_bit_cast(bf16x8, As[fa[ks] + mi * FSTR]);
#pragma unroll
            for (int ni = 0; ni < NI; ++ni)
                xb[b][ni] = __builtin_bit_cast(bf16x8, Bs[fb[ks] + ni * FSTR]);
        };
        read(0, 0);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            if (ks + 1 < KS)
                read(ks + 1, (ks + 1) & 1);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int mi = 0; mi < MI; ++mi)
#pragma unroll
                for (int ni = 0; ni < NI; ++ni)
                    acc[mi][ni] = Op::run(xa[ks & 1][mi], xb[ks & 1][ni], acc[mi][ni]);
            __builtin_amdgcn_sched_barrier(0);
            after(ks);
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    const int nst = (p.KC + CH - 1) / CH;
    if (nst > 0)
        issue(0, A0, B0);
    if (NS > 2 && nst > 1)
        issue(1, A1, B1);
    for (int s0 = 0; s0 < nst; s0 += NS) {
#pragma unroll
        for (int h = 0; h < NS; ++h) {
            const int s = s0 + h;
            if (s >= nst)
                break;
            u32x4* Ac = h == 0 ? A0 : (h == 1 ? A1 : A2);
            u32x4* Bc = h == 0 ? B0 : (h == 1 ? B1 : B2);
            const int hnx = (h + NS - 1) % NS;
            u32x4* An = hnx == 0 ? A0 : (hnx == 1 ? A1 : A2);
            u32x4* Bn = hnx == 0 ? B0 : (hnx == 1 ? B1 : B2);
            if (NS > 2 && s + 1 < nst)
                wait_all_but_next();
            else
                wait_vmcnt<0>();
            stage_barrier();
            // one code path: the copies of stage t are skipped (a uniform
            // branch) past the last stage
            const int t = s + NS - 1;
            const bool more = t < nst;
            const uint32_t d = b_delta(t);
            compute(Ac, Bc, [&](int part) {
                if (more)
                    issue_part(t, An, Bn, part, d);
            });
        }
    }

    const int brow = wn * NI * MT + lane % MT;

    // ---- epilogue (branch-free: masked lanes store to an out-of-range offset)
    const __amdgpu_buffer_rsrc_t ry = make_rsrc(p.Y, p.Y_bytes);
    if constexpr (EPI == 0) {
        int cbase[NI];
        uint32_t cbad[NI];
#pragma unroll
        for (int ni = 0; ni < NI; ++ni) {
            const int col = n0 + brow + ni * MT;
            const int n = (int)fdiv((uint32_t)col, p.div_ohw);
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
    } else if constexpr (EPI == 2) {
        // The data gradient as the layer below's staged top gradient (stride
        // 1: the GEMM's column grid is the image, row m is channel
        // g*Cg_out + m) and the bias gradient's partial sums of each wave's
        // 64 columns.  A lane holds four consecutive channels of one pixel
        // per register quad: one 8-byte store.
        static_assert(MT == 32 && WN == 4 && NI * MT == 64, "stage-below epilogue layout");
        const int OutHW = p.OutH * p.OutW;
        const __amdgpu_buffer_rsrc_t rom =
            make_rsrc(p.Omask, MASK == 1 ? p.Y_bytes / 2 : (MASK == 2 ? p.Y_bytes : 0u));
        const __amdgpu_buffer_rsrc_t rsh = make_rsrc(p.Sh, p.Sh_bytes);
        const __amdgpu_buffer_rsrc_t rss = make_rsrc(p.Ssum, p.Ssum_bytes);
        int mb[NI], sb[NI];
        uint32_t pbad[NI];
#pragma unroll
        for (int ni = 0; ni < NI; ++ni) {
            const int col = n0 + brow + ni * MT;
            const bool cok = col < p.Ncol;
            const int n = cok ? (int)fdiv((uint32_t)col, p.div_ohw) : 0;
            const int pix = col - n * OHW;
            const int a = (int)fdiv((uint32_t)pix, p.div_ow);
            const int b = pix - a * p.OW;
            const int h = a + p.a0h - p.oph, w = b + p.a0w - p.opw;
            const bool ok = cok && (unsigned)h < (unsigned)p.OutH && (unsigned)w < (unsigned)p.OutW;
            pbad[ni] = ok ? 0u : kOob;
            mb[ni] = (n * p.Cout + g * p.Cg_out) * OutHW + h * p.OutW + w;
            sb[ni] = ((n * p.s_Hp + h + p.s_tb) * p.s_Wp + w + p.s_lb) * p.s_Ktot + g * p.Cg_out;
        }
        const int lrow0 = m0 + wm * MI * MT;
#pragma unroll
        for (int mi = 0; mi < MI; ++mi) {
            // the mask values of the block first, then the values and stores
            float y[Op::kRegs][NI];
#pragma unroll
            for (int q = 0; q < Op::kRegs; ++q) {
                const int m = lrow0 + mi * MT + Op::row(q, lane);
#pragma unroll
                for (int ni = 0; ni < NI; ++ni) {
                    const uint32_t bad = pbad[ni] | ((uint32_t)(m >= M) << 31);
                    const uint32_t idx = (uint32_t)(mb[ni] + m * OutHW);
                    if constexpr (MASK == 1)
                        y[q][ni] = bf16_to_f32(buf_ld_u16(rom, (idx * 2u) | bad));
                    else if constexpr (MASK == 2)
                        y[q][ni] = buf_ld_f32(rom, (idx * 4u) | bad);
                    else
                        y[q][ni] = 1.f;
                }
            }
#pragma unroll
            for (int qa = 0; qa < Op::kRegs / 4; ++qa) {
                float csum[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ni = 0; ni < NI; ++ni) {
                    float vq[4];
#pragma unroll
                    for (int b = 0; b < 4; ++b) {
                        const int q = 4 * qa + b;
                        float v = acc[mi][ni][q];
                        if constexpr (MASK == 1)
                            v = y[q][ni] > 0.f ? v : 0.f;
                        else if constexpr (MASK == 2)
                            v = y[q][ni] > 0x1p-134f ? v : 0.f;
                        // (positions outside the image add nothing)
                        v = pbad[ni] ? 0.f : v;
                        csum[b] += v;
                        vq[b] = v;
                    }
                    const uint32_t w2[2] = {f32x2_to_bf16x2_rne(vq[0], vq[1]),
                                            f32x2_to_bf16x2_rne(vq[2], vq[3])};
                    // rows m .. m + 3 of this quad; a quad past M stores nothing
                    const int m = lrow0 + mi * MT + Op::row(4 * qa, lane);
                    const uint32_t off = ((uint32_t)(sb[ni] + m) * 2u) | pbad[ni] |
                                         ((uint32_t)(m >= M) << 31);
                    __builtin_amdgcn_raw_buffer_store_b64(u32x2{w2[0], w2[1]}, rsh, off, 0, 0);
                }
                // the wave's column sums: over the 32 lanes of each half
#pragma unroll
                for (int b = 0; b < 4; ++b) {
                    float t = csum[b];
#pragma unroll
                    for (int o = 16; o > 0; o >>= 1)
                        t += __shfl_xor(t, o, 64);
                    const int m = lrow0 + mi * MT + Op::row(4 * qa + b, lane);
                    const uint32_t off =
                        ((uint32_t)((g * p.Cg_out + m) * p.s_T + 4 * ct + wn) * 4u) |
                        ((uint32_t)((lane & 31) != 0 || m >= M) << 31);
                    buf_st_f32(t, rss, off);
                }
            }
        }
    } else {
        const int pss = p.psh * p.psw;
        const int OutHW = p.OutH * p.OutW;
        // the bottom mask (MASK 1: bf16 values, MASK 2: float values taken
        // as the bf16 they round to)
        const __amdgpu_buffer_rsrc_t rom =
            make_rsrc(p.Omask, MASK == 1 ? p.Y_bytes / 2 : (MASK == 2 ? p.Y_bytes : 0u));
        int cb[NI], hb[NI], wb[NI];
#pragma unroll
        for (int ni = 0; ni < NI; ++ni) {
            const int col = n0 + brow + ni * MT;
            const bool cok = col < p.Ncol;
            const int n = cok ? (int)fdiv((uint32_t)col, p.div_ohw) : 0;
            const int pix = col - n * OHW;
            const int a = (int)fdiv((uint32_t)pix, p.div_ow);
            const int b = pix - a * p.OW;
            hb[ni] = cok ? p.psh * (a + p.a0h) - p.oph : -(1 << 28);
            wb[ni] = p.psw * (b + p.a0w) - p.opw;
            cb[ni] = (n * p.Cout + g * p.Cg_out) * OutHW;
        }
        // per MT-row block: every position (and, masked, every bf16 bottom
        // value) first, then the stores (a load after a store to another
        // buffer could not be moved above it, so each would wait alone)
#pragma unroll
        for (int mi = 0; mi < MI; ++mi) {
            uint32_t off[Op::kRegs][NI];
            float y[Op::kRegs][NI];
#pragma unroll
            for (int q = 0; q < Op::kRegs; ++q) {
                const int m = m0 + wm * MI * MT + mi * MT + Op::row(q, lane);
                int c = m, fh = 0, fw = 0;
                if (pss != 1) {
                    c = (int)fdiv((uint32_t)m, p.div_pss);
                    const int fr = m - c * pss;
                    fh = (int)fdiv((uint32_t)fr, p.div_psw);
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
                    off[q][ni] = idx | bad;
                    // backward of the ReLU whose (bf16) output is this
                    // layer's bottom: keep the gradient where it was > 0
                    if constexpr (MASK == 1)
                        y[q][ni] = bf16_to_f32(buf_ld_u16(rom, (idx * 2u) | bad));
                    else if constexpr (MASK == 2)
                        y[q][ni] = buf_ld_f32(rom, (idx * 4u) | bad);
                }
            }
#pragma unroll
            for (int q = 0; q < Op::kRegs; ++q)
#pragma unroll
                for (int ni = 0; ni < NI; ++ni) {
                    float v = acc[mi][ni][q];
                    // (a float rounds to a positive bf16 exactly when it is
                    // above 2^-134, the tie that rounds to even 0; NaN never)
                    if constexpr (MASK == 1)
                        v = y[q][ni] > 0.f ? v : 0.f;
                    else if constexpr (MASK == 2)
                        v = y[q][ni] > 0x1p-134f ? v : 0.f;
                    const uint32_t o = off[q][ni];
                    buf_st_f32(v, ry, ((o & ~kOob) * 4u) | (o & kOob));
                }
        }
    }
}

// ----------------------------------------------------------- weight gradient
// Split-K over the output pixels (n, i, j), TKP = 64 per stage.  Both operands
// are gathered pixel by pixel into LDS tiles laid out [pixel][channel] (the
// channel-contiguous staging read as is): a pixel row of the D tile holds the
// tile's 128 output channels, one of the X tile the tile's TN reduction
// indices r = (u, v, c) (8 channels of one tap per 16-byte chunk), each
// 64-channel line of a row copied by 16-byte DMA as in the forward kernel
// (8 rows x 128 bytes per wave copy, chunks swizzled by chunk_swz of the
// pixel).  The instructions want 8 consecutive pixels per lane for one
// channel; ds_read_b64_tr_b16 supplies them: in each group of 16 lanes, lane
// (4i + q) points at channels 4q .. 4q + 3 of pixel row k0 + i, and lane j of
// the group receives pixels k0 .. k0 + 3 of channel j.  Two such reads make a
// fragment.
typedef short short4v __attribute__((ext_vector_type(4)));

__device__ __forceinline__ short4v lds_read_tr16(const void* p)
{
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) short4v*)p);
}

// Byte offset of element (pixel k, channel c) in a [pixel][channel] tile of
// NL 64-channel lines per pixel.
__device__ __forceinline__ int wtile_off(int k, int c, int NL)
{
    return ((k >> 3) * NL + (c >> 6)) * 1024 + (k & 7) * 128 +
           ((((c & 63) >> 3) ^ chunk_swz(k)) << 4) + (c & 7) * 2;
}

template <int WM, int WN, int MI, int NI, int NS>
__global__ void __launch_bounds__(64 * WM * WN)
conv_wgrad_bf16_kernel(const WgradBf16Params p)
{
    constexpr int MT = 32;
    constexpr int NW = WM * WN;
    constexpr int TM = WM * MI * MT;
    constexpr int TN = WN * NI * MT;
    constexpr int TKP = 64;            // pixels per stage
    constexpr int KS = TKP / 16;       // instructions along k per stage
    constexpr int NLA = 2;             // 64-channel lines per D row (TM <= 128)
    constexpr int NLB = TN / 64;       // lines per X row
    constexpr int EA = TKP / 8 / NW;   // row groups (8 pixels) per wave
    constexpr int NC = EA * (NLA + NLB);
    constexpr int CPP = (NC + KS - 1) / KS;
    static_assert((NW == 4 || NW == 8) && TM <= 128 && TN % 64 == 0 && EA * NW * 8 == TKP,
                  "tile shape");
    static_assert(NS == 2 || NS == 3, "buffers");

    __shared__ u32x4 A0[TKP * NLA * 8], A1[TKP * NLA * 8], A2[NS > 2 ? TKP * NLA * 8 : 1];
    __shared__ u32x4 B0[TKP * NLB * 8], B1[TKP * NLB * 8], B2[NS > 2 ? TKP * NLB * 8 : 1];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave % WM;
    const int wn = wave / WM;
    const int n_rt = (p.Rw + TN - 1) / TN;
    const int n_mt = (p.Kg + TM - 1) / TM;
    int T = blockIdx.x;
    if (p.unit_order) {
        // workgroups are dealt round-robin over the 8 XCDs: slot s of XCD x
        // takes block s % U of unit (s / U) * 8 + x
        const int U = n_rt * n_mt;
        const int slot = blockIdx.x >> 3;
        const int unit = (slot / U) * 8 + (blockIdx.x & 7);
        T = unit * U + slot % U;
    }
    if (T >= n_rt * n_mt * p.G * p.splits)
        return;
    const int rt = T % n_rt;
    const int mt = (T / n_rt) % n_mt;
    const int g = (T / (n_rt * n_mt)) % p.G;
    const int split = T / (n_rt * n_mt * p.G);
    const int m0 = mt * TM;
    const int r0 = rt * TN;
    const int OHW = p.OH * p.OW;
    const int col_begin = split * p.cols_per_split;
    const int col_end = min(p.Ncol, col_begin + p.cols_per_split);

    const __amdgpu_buffer_rsrc_t rd = make_rsrc(p.D, p.D_bytes);
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(p.X, p.X_bytes);

    // copies: this wave's row groups EA*wave + e (pixels 8*(EA*wave + e) +
    // lane/8 of a stage), lane's chunk of a line (lane % 8) ^ chunk_swz(pixel).  Byte
    // offsets from a pixel: rows past Kg and columns past Rw are read (inside
    // the buffer or as zeros past its end) but feed only results that are
    // never stored, so they need no mask.
    const int cr = lane >> 3;
    uint32_t a_off[EA][NLA], b_off[EA][NLB];
#pragma unroll
    for (int e = 0; e < EA; ++e) {
        const int ch = (lane & 7) ^ chunk_swz(8 * (EA * wave + e) + cr);
#pragma unroll
        for (int L = 0; L < NLA; ++L)
            a_off[e][L] = (uint32_t)(g * p.Kgp + m0 + 64 * L + 8 * ch) * 2u;
#pragma unroll
        for (int L = 0; L < NLB; ++L) {
            const int r = r0 + 64 * L + 8 * ch;  // 8 channels of one tap
            const int t = r / p.Cgp;
            const int c = r - t * p.Cgp;
            const int u = t / p.kw;
            const int v = t - u * p.kw;
            b_off[e][L] = (uint32_t)((u * p.IWp + v) * p.Ctot + g * p.Cgp + c) * 2u;
        }
    }
    // byte offsets of this wave's pixel rows in stage t; kOob past the
    // split's end (base + offset then stays out of range: offsets < 2^31)
    uint32_t pd[EA], px[EA];
    auto pixels = [&](int t) {
#pragma unroll
        for (int e = 0; e < EA; ++e) {
            const int col = col_begin + t * TKP + 8 * (EA * wave + e) + cr;
            const int n = (int)fdiv((uint32_t)col, p.div_ohw);
            const int pix = col - n * OHW;
            const int i = (int)fdiv((uint32_t)pix, p.div_ow);
            const int j = pix - i * p.OW;
            const bool ok = col < col_end;
            pd[e] = ok ? (uint32_t)(((n * p.DHp + i + p.dtb) * p.DWp + j + p.dlb) * p.Ktot) * 2u
                       : kOob;
            px[e] = ok ? (uint32_t)(((n * p.IHp + i * p.sh) * p.IWp + j * p.sw) * p.Ctot) * 2u
                       : kOob;
        }
    };
    auto issue_part = [&](u32x4* As, u32x4* Bs, int part) {
#pragma unroll
        for (int c = part * CPP; c < (part + 1) * CPP && c < NC; ++c) {
            const int e = c / (NLA + NLB);
            const int L = c % (NLA + NLB);
            const int rg = EA * wave + e;
            if (L < NLA)
                copy16_lds(rd, &As[(rg * NLA + L) * 64], pd[e] + a_off[e][L], 0u);
            else
                copy16_lds(rx, &Bs[(rg * NLB + L - NLA) * 64], px[e] + b_off[e][L - NLA], 0u);
        }
    };
    auto issue = [&](int t, u32x4* As, u32x4* Bs) {
        pixels(t);
#pragma unroll
        for (int part = 0; part < KS; ++part)
            issue_part(As, Bs, part);
    };
    auto wait_all_but_next = [&]() { wait_vmcnt<NC>(); };

    floatx16 acc[MI][NI];
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int ni = 0; ni < NI; ++ni)
            acc[mi][ni] = floatx16{};

    // transposed-read addresses: lane as a source points at pixel
    // 8*(lane/32) + 4h + (lane%16)/4 of the step, channel 16*((lane/16)%2) +
    // 4*(lane%4) of its 32-row block; steps ks add 16 pixels (2 row groups)
    const int ksrc = 8 * (lane >> 5) + ((lane & 15) >> 2);
    const int csrc = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
    int fa[MI][2], fb[NI][2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
#pragma unroll
        for (int mi = 0; mi < MI; ++mi)
            fa[mi][h] = wtile_off(ksrc + 4 * h, wm * MI * MT + mi * MT + csrc, NLA);
#pragma unroll
        for (int ni = 0; ni < NI; ++ni)
            fb[ni][h] = wtile_off(ksrc + 4 * h, wn * NI * MT + ni * MT + csrc, NLB);
    }

    auto compute = [&](const u32x4* As, const u32x4* Bs, auto&& after) {
        const char* a = (const char*)As;
        const char* b = (const char*)Bs;
        bf16x8 xa[2][MI], xb[2][NI];
        auto read = [&](int ks, int buf) {
#pragma unroll
            for (int mi = 0; mi < MI; ++mi) {
                const short4v lo = lds_read_tr16(a + fa[mi][0] + ks * 2 * NLA * 1024);
                const short4v hi = lds_read_tr16(a + fa[mi][1] + ks * 2 * NLA * 1024);
                xa[buf][mi] = __builtin_bit_cast(
                    bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
            }
#pragma unroll
            for (int ni = 0; ni < NI; ++ni) {
                const short4v lo = lds_read_tr16(b + fb[ni][0] + ks * 2 * NLB * 1024);
                const short4v hi = lds_read_tr16(b + fb[ni][1] + ks * 2 * NLB * 1024);
                xb[buf][ni] = __builtin_bit_cast(
                    bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
            }
        };
        read(0, 0);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            if (ks + 1 < KS)
                read(ks + 1, (ks + 1) & 1);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int mi = 0; mi < MI; ++mi)
#pragma unroll
                for (int ni = 0; ni < NI; ++ni)
                    acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        xa[ks & 1][mi], xb[ks & 1][ni], acc[mi][ni], 0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
            after(ks);
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    const int nst = col_end > col_begin ? (col_end - col_begin + TKP - 1) / TKP : 0;
    if (nst > 0)
        issue(0, A0, B0);
    if (NS > 2 && nst > 1)
        issue(1, A1, B1);
    for (int s0 = 0; s0 < nst; s0 += NS) {
#pragma unroll
        for (int h = 0; h < NS; ++h) {
            const int s = s0 + h;
            if (s >= nst)
                break;
            u32x4* Ac = h == 0 ? A0 : (h == 1 ? A1 : A2);
            u32x4* Bc = h == 0 ? B0 : (h == 1 ? B1 : B2);
            const int hnx = (h + NS - 1) % NS;
            u32x4* An = hnx == 0 ? A0 : (hnx == 1 ? A1 : A2);
            u32x4* Bn = hnx == 0 ? B0 : (hnx == 1 ? B1 : B2);
            if (NS > 2 && s + 1 < nst)
                wait_all_but_next();
            else
                wait_vmcnt<0>();
            stage_barrier();
            const int t = s + NS - 1;
            const bool more = t < nst;
            if (more)
                pixels(t);
            compute(Ac, Bc, [&](int part) {
                if (more)
                    issue_part(An, Bn, part);
            });
        }
    }

    // Partial result P[split][g*Kg + m][r], lanes along r
    const __amdgpu_buffer_rsrc_t rp = make_rsrc(p.P, p.P_bytes);
    const int pbase = split * p.K * p.Rw;
#pragma unroll
    for (int ni = 0; ni < NI; ++ni) {
        const int r = r0 + wn * NI * MT + ni * MT + (lane & 31);
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

// dW[k][c][u][v] = (accumulate ? dW : 0) + sum_s P[s][k][(bu*kwp + bv)*Cgp + cp]
// (c < Cg, u < kh, v < kw): the split partials added in a fixed order, as
// wgrad_reduce_kernel does, with lanes along the partials' (bu, bv, cp)
// order.  Plain staging (S = 1): (bu, bv, cp) = (u, v, c).  Space-to-depth
// staging by S: u = S*bu + fu, v = S*bv + fv, cp = (fu*S + fv)*Cg + c.
constexpr int kPermParts = 8;
constexpr int kPermCols = 32;

__global__ void __launch_bounds__(kPermParts * kPermCols)
wgrad_reduce_perm_kernel(const float* __restrict__ P, float* __restrict__ dW, int K, int Rw,
                         int Cgp, int Cg, int kh, int kw, int kwp, int S, int splits,
                         int accumulate)
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
        const int cp = r - tap * Cgp;
        const int bu = tap / kwp;
        const int bv = tap - bu * kwp;
        const int f = cp / Cg;
        const int c = cp - f * Cg;
        const int fu = f / S;
        const int u = S * bu + fu;
        const int v = S * bv + f - fu * S;
        if (f < S * S && u < kh && v < kw) {
            float* o = dW + (((size_t)k * Cg + c) * kh + u) * kw + v;
            *o = accumulate ? *o + t : t;
        }
    }
}

// ------------------------------------------------------------------ staging
// NCHW bf16 -> zero-bordered channel-contiguous bf16 with per-group channel
// padding, through a CT-channel x PT-pixel LDS tile (CT = 8 .. 64, sized to
// the padded channel count; PT = min(4096 / CT, 256)) over the bordered
// Hp x Wp grid: coalesced 2-byte reads along pixels (zeros outside the
// image), 16-byte writes along channels.
template <int CT>
constexpr int stage_tile_pixels()
{
    return 4096 / CT < 256 ? 4096 / CT : 256;
}

// A staged value: bf16 as given, or a float rounded to nearest-even.
__device__ __forceinline__ bf16_t to_bf16(bf16_t v) { return v; }
__device__ __forceinline__ bf16_t to_bf16(float v) { return f32_to_bf16_rne(v); }
// two staged values packed, the first in the low half
__device__ __forceinline__ uint32_t to_bf16x2(bf16_t a, bf16_t b)
{
    return (uint32_t)a | ((uint32_t)b << 16);
}
__device__ __forceinline__ uint32_t to_bf16x2(float a, float b) { return f32x2_to_bf16x2_rne(a, b); }

// Row-chunk staging (groups of a multiple of 8 channels, so that Cgp = Cg and
// the staged channels are the blob's; rows of at most kStageRowPixels pixels):
// a block takes image n, channels c0 .. c0 + 63 and padded rows
// r0 .. r0 + RH - 1.  The real rows among them are one contiguous run of
// RP = rows * W pixels in every channel plane, so the loads are whole runs,
// one pixel per thread and channel (no line is shared with another block but
// at the run's ends); the block transposes them through LDS and writes every
// padded pixel of its rows, border zeros included, as 16-byte chunks of 8
// channels.
constexpr int kStageRowPixels = 256;

template <typename T>
__device__ __forceinline__ T load_elem(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff);
template <>
__device__ __forceinline__ float load_elem<float>(__amdgpu_buffer_rsrc_t r, uint32_t voff,
                                                  uint32_t soff)
{
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0));
}
template <>
__device__ __forceinline__ bf16_t load_elem<bf16_t>(__amdgpu_buffer_rsrc_t r, uint32_t voff,
                                                    uint32_t soff)
{
    return __builtin_amdgcn_raw_buffer_load_b16(r, voff, soff, 0);
}
constexpr int kStageRowCh = 64;

template <typename T>
__global__ void __launch_bounds__(256)
stage_rows_bf16_kernel(const T* __restrict__ X, bf16_t* __restrict__ Xp, int C, int H, int W,
                       int Cg, int Cgp, int Ctot, int Hp, int Wp, int tb, int lb, int RH,
                       int rchunks, int ctiles)
{
    constexpr int CT = kStageRowCh;
    constexpr int C8 = CT / 8;
    __shared__ bf16_t tile[CT][kStageRowPixels + 2];
    // block -> (n, channel tile, row chunk), row chunks fastest
    const int n = blockIdx.x / (rchunks * ctiles);
    const int rem = blockIdx.x - n * rchunks * ctiles;
    const int ct = rem / rchunks;
    const int r0 = (rem - ct * rchunks) * RH;
    const int r1 = min(Hp, r0 + RH);
    const int c0 = ct * CT;
    const int h0 = max(0, r0 - tb);
    const int h1 = min(H, r1 - tb);
    const int RP = h1 > h0 ? (h1 - h0) * W : 0;
    const int tid = threadIdx.x;
    if (tid < RP) {
        // the image's planes through one buffer resource: channel c0 + c is
        // the scalar offset (c0 + c) * H * W elements, out of range (0) past
        // the last channel
        const uint32_t plane = (uint32_t)(H * W) * (uint32_t)sizeof(T);
        const __amdgpu_buffer_rsrc_t rx =
            make_rsrc(X + (size_t)n * C * H * W, (uint32_t)C * plane);
        const uint32_t voff = (uint32_t)(h0 * W + tid) * (uint32_t)sizeof(T);
        // every load of the thread in flight before the first is used
        T v[CT];
#pragma unroll
        for (int c = 0; c < CT; ++c)
            v[c] = load_elem<T>(rx, voff, (uint32_t)(c0 + c) * plane);
#pragma unroll
        for (int c = 0; c < CT; ++c)
            tile[c][tid] = to_bf16(v[c]);
    }
    __syncthreads();
    const int npix = (r1 - r0) * Wp;
    for (int id = tid; id < npix * C8; id += 256) {
        const int c8 = id % C8;
        const int pl = id / C8;
        const int cp = c0 + 8 * c8;
        if (cp >= Ctot)
            continue;
        const int hp = r0 + pl / Wp;
        const int wp = pl - (pl / Wp) * Wp;
        const int h = hp - tb;
        const int w = wp - lb;
        u32x4 out = {0u, 0u, 0u, 0u};
        if ((unsigned)h < (unsigned)H && (unsigned)w < (unsigned)W) {
            const int q = (h - h0) * W + w;
#pragma unroll
            for (int k = 0; k < 4; ++k)
                out[k] = (uint32_t)tile[8 * c8 + 2 * k][q] |
                         ((uint32_t)tile[8 * c8 + 2 * k + 1][q] << 16);
        }
        *(u32x4*)&Xp[(((size_t)n * Hp + hp) * Wp + wp) * Ctot + cp] = out;
    }
}

template <int CT, typename T>
__global__ void __launch_bounds__(256)
stage_nhwc_bf16_kernel(const T* __restrict__ X, bf16_t* __restrict__ Xp, int C, int H, int W,
                       int Cg, int Cgp, int Ctot, int Hp, int Wp, int tb, int lb, int ptiles,
                       int ctiles)
{
    constexpr int PT = stage_tile_pixels<CT>();
    constexpr int C8 = CT / 8;
    constexpr int NQ = CT * PT / 256;  // tile elements per thread
    constexpr int NW = PT * C8 / 256;  // 16-byte writes per thread
    static_assert(256 % PT == 0 && NW >= 1, "tile shape");
    __shared__ bf16_t tile[CT][PT + 2];
    // block -> (n, channel tile, pixel tile), pixel tiles fastest
    const int n = blockIdx.x / (ptiles * ctiles);
    const int rem = blockIdx.x - n * ptiles * ctiles;
    const int ct = rem / ptiles;
    const int c0 = ct * CT;
    const int p0 = (rem - ct * ptiles) * PT;
    const int HWp = Hp * Wp;
    const int tid = threadIdx.x;
    // the thread's pixel is the same for every element it loads (256 % PT == 0)
    const int px = tid % PT;
    const int pix = p0 + px;
    const int hp = pix / Wp;
    const int h = hp - tb;
    const int w = pix - hp * Wp - lb;
    const bool inside = pix < HWp && (unsigned)h < (unsigned)H && (unsigned)w < (unsigned)W;
    const size_t src = (size_t)n * C * H * W + (size_t)h * W + w;
    // all of the thread's loads are issued before the first LDS store
    bf16_t v[NQ];
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
        const int c = (tid + 256 * q) / PT;
        const int cp = c0 + c;
        const int g = cp / Cgp;
        const int cl = cp - g * Cgp;
        v[q] = inside && cp < Ctot && cl < Cg ? to_bf16(X[src + (size_t)(g * Cg + cl) * H * W])
                                              : (bf16_t)0;
    }
#pragma unroll
    for (int q = 0; q < NQ; ++q)
        tile[(tid + 256 * q) / PT][px] = v[q];
    __syncthreads();
#pragma unroll
    for (int q = 0; q < NW; ++q) {
        const int id = tid + 256 * q;
        const int pl = id / C8;
        const int c8 = id % C8;
        const int pw = p0 + pl;
        const int cp = c0 + 8 * c8;
        if (pw < HWp && cp < Ctot) {
            u32x4 v;
#pragma unroll
            for (int k = 0; k < 4; ++k)
                v[k] = (uint32_t)tile[8 * c8 + 2 * k][pl] |
                       ((uint32_t)tile[8 * c8 + 2 * k + 1][pl] << 16);
            *(u32x4*)&Xp[((size_t)n * HWp + pw) * Ctot + cp] = v;
        }
    }
}

// NCHW bf16 -> zero-bordered pixel-interleaved bf16 for one group of Cgp = 1,
// 2 or 4 channels (c < Cg real, the rest 0): thread q writes the 16-byte
// chunk of padded pixels TPC*q .. TPC*q + TPC - 1 (TPC = 8 / Cgp; Hp*Wp is a
// multiple of TPC), its lanes reading consecutive pixel groups of each plane.
template <int CGP, typename T>
__global__ void __launch_bounds__(256)
stage_narrow_bf16_kernel(const T* __restrict__ X, bf16_t* __restrict__ Xp, int Cg, int H, int W,
                         int Hp, int Wp, int tb, int lb, FastDiv div_wp)
{
    constexpr int TPC = 8 / CGP;
    // grid: x over the image's chunks, y over the images
    const int n = blockIdx.y;
    const int per_image = Hp * Wp / TPC;
    const int q = blockIdx.x * 256 + threadIdx.x;
    if (q >= per_image)
        return;
    // the image's planes through one buffer resource: channel c is the
    // scalar offset c * H * W elements, out of range (0) from channel Cg on,
    // and a pixel outside the image takes the out-of-range lane offset
    const uint32_t plane = (uint32_t)(H * W) * (uint32_t)sizeof(T);
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(X + (size_t)n * Cg * H * W, (uint32_t)Cg * plane);
    T v[TPC][CGP];
#pragma unroll
    for (int t = 0; t < TPC; ++t) {
        const int pix = q * TPC + t;
        const int hp = (int)fdiv((uint32_t)pix, div_wp);
        const int h = hp - tb;
        const int x = pix - hp * Wp - lb;
        const bool inside = (unsigned)h < (unsigned)H && (unsigned)x < (unsigned)W;
        const uint32_t voff = inside ? (uint32_t)(h * W + x) * (uint32_t)sizeof(T) : kOob;
#pragma unroll
        for (int c = 0; c < CGP; ++c)
            v[t][c] = load_elem<T>(rx, voff, (uint32_t)c * plane);
    }
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 8; e += 2)  // elements e, e + 1 of the chunk: (tap, channel) pairs
        w[e >> 1] = to_bf16x2(v[e / CGP][e % CGP], v[(e + 1) / CGP][(e + 1) % CGP]);
    *(u32x4*)&Xp[((size_t)n * per_image + q) * 8] = u32x4{w[0], w[1], w[2], w[3]};
}

// Top-gradient staging: Dh = bf16(relu ? G [Y > 0] : G) channel-contiguous on
// the zero-bordered Hp x Wp grid.  One block per (image, 64 padded channels,
// run of kDiffPrepPixels bordered pixels), walking its run 64 pixels at a
// time: each thread loads one pixel of 16 channels (all loads of a step
// issued before any is used), the block transposes them through LDS and
// writes 16-byte channel chunks.  Each thread also adds up the fp32 masked
// gradient of its 16 channels; one wave sum per channel at the end (a fixed
// butterfly after a fixed per-lane order; the border adds 0) gives
// sums[(g*Kg + k) * T + n * runs + run] (T = N * runs), the partial
// bias gradient of that run of the image.
constexpr int kDiffPrepPixels = 512;

template <bool RELU>
__global__ void __launch_bounds__(256)
diff_prep_bf16_kernel(const float* __restrict__ G, const float* __restrict__ Y,
                      bf16_t* __restrict__ Dh, float* __restrict__ sums, int N, int K, int H,
                      int W, int Kg, int Kgp, int Ktot, int Hp, int Wp, int tb, int lb,
                      int ctiles, int runs)
{
    constexpr bool relu = RELU;
    __shared__ bf16_t tile[64][66];
    const int run = blockIdx.x % runs;
    const int nc = blockIdx.x / runs;
    const int n = nc / ctiles;
    const int c0 = (nc - n * ctiles) * 64;
    const int HWp = Hp * Wp;
    const int p_begin = run * kDiffPrepPixels;
    const int p_end = min(HWp, p_begin + kDiffPrepPixels);
    const int tid = threadIdx.x;
    const int px = tid & 63;
    const int cw = tid >> 6;
    const int plane = H * W;
    // G and Y through buffer resources (both < 2^31 bytes): a missing channel
    // or a border pixel is an out-of-range offset and reads 0
    const uint32_t gbytes = (uint32_t)((size_t)N * K * plane * 4);
    const __amdgpu_buffer_rsrc_t rg = make_rsrc(G, gbytes);
    const __amdgpu_buffer_rsrc_t ry = make_rsrc(Y, RELU ? gbytes : 0u);
    // this thread's 16 channels (cw + 4q): byte offsets of their planes,
    // 2^31 for a channel that does not exist
    uint32_t cb4[16];
    bool cok[16];
#pragma unroll
    for (int q = 0; q < 16; ++q) {
        const int cp = c0 + cw + 4 * q;
        const int g = cp / Kgp;
        const int k = cp - g * Kgp;
        cok[q] = cp < Ktot && k < Kg;
        cb4[q] = cok[q] ? (uint32_t)((n * K + g * Kg + k) * plane) * 4u : kOob;
    }
    float acc[16];
#pragma unroll
    for (int q = 0; q < 16; ++q)
        acc[q] = 0.f;
    // the byte offset of this thread's pixel in step p0 (out of range on the
    // border and past the run)
    auto step_off = [&](int p0) -> uint32_t {
        const int pix = p0 + px;
        const int hp = pix / Wp;
        const int h = hp - tb;
        const int w = pix - hp * Wp - lb;
        const bool inside = pix < p_end && (unsigned)h < (unsigned)H && (unsigned)w < (unsigned)W;
        return inside ? (uint32_t)(h * W + w) * 4u : kOob;
    };
    // Each step's loads go out before the previous step is transposed and
    // stored (two steps in flight per thread); the ReLU output's too.
    float d[16], y[16];
    {
        const uint32_t o = step_off(p_begin);
#pragma unroll
        for (int q = 0; q < 16; ++q)
            d[q] = buf_ld_f32(rg, (cb4[q] + o) | (o & kOob));
        if constexpr (RELU) {
#pragma unroll
            for (int q = 0; q < 16; ++q)
                y[q] = buf_ld_f32(ry, (cb4[q] + o) | (o & kOob));
        }
    }
    for (int p0 = p_begin; p0 < p_end; p0 += 64) {
        float dn[16], yn[16];
        const bool more = p0 + 64 < p_end;
        if (more) {
            const uint32_t o = step_off(p0 + 64);
#pragma unroll
            for (int q = 0; q < 16; ++q)
                dn[q] = buf_ld_f32(rg, (cb4[q] + o) | (o & kOob));
            if constexpr (RELU) {
#pragma unroll
                for (int q = 0; q < 16; ++q)
                    yn[q] = buf_ld_f32(ry, (cb4[q] + o) | (o & kOob));
            }
        }
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            // (a NaN output masks too)
            const float v = !relu || y[q] > 0.f ? d[q] : 0.f;
            acc[q] += v;
            tile[cw + 4 * q][px] = f32_to_bf16_rne(v);
        }
        __syncthreads();
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const int id = tid + 256 * q;
            const int pl = id >> 3;
            const int c8 = id & 7;
            const int pw = p0 + pl;
            const int cp = c0 + 8 * c8;
            if (pw < p_end && cp < Ktot) {
                u32x4 v;
#pragma unroll
                for (int k = 0; k < 4; ++k)
                    v[k] = (uint32_t)tile[8 * c8 + 2 * k][pl] |
                           ((uint32_t)tile[8 * c8 + 2 * k + 1][pl] << 16);
                *(u32x4*)&Dh[((size_t)n * HWp + pw) * Ktot + cp] = v;
            }
        }
        __syncthreads();
        if (more) {
#pragma unroll
            for (int q = 0; q < 16; ++q) {
                d[q] = dn[q];
                if constexpr (RELU)
                    y[q] = yn[q];
            }
        }
    }
    if (sums) {
        const size_t T = (size_t)N * runs;
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            const float sm = wave_sum(acc[q]);
            if (px == 0 && cok[q]) {
                const int cp = c0 + cw + 4 * q;
                const int g = cp / Kgp;
                sums[(size_t)(g * Kg + cp - g * Kgp) * T + (size_t)n * runs + run] = sm;
            }
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

// Forward weights in the staged reduction order, rows padded to Rp:
// Wp[o][(bu*kwp + bv)*Cgp + cp] = W[o][c][u][v] with (u, v, c) as in
// wgrad_reduce_perm_kernel (S = 1: (bu, bv, cp) = (u, v, c)), zero where u, v
// or c falls outside the kernel or the channels and for r >= the staged taps.
__global__ void __launch_bounds__(256)
pack_weights_bf16_kernel(const bf16_t* __restrict__ W, bf16_t* __restrict__ Wp, int K, int Cg,
                         int Cgp, int kh, int kw, int kwp, int S, int Rp)
{
    const long total = (long)K * Rp;
    for (long e = blockIdx.x * (long)blockDim.x + threadIdx.x; e < total;
         e += (long)gridDim.x * blockDim.x) {
        const int o = (int)(e / Rp);
        const int r = (int)(e - (long)o * Rp);
        const int t = r / Cgp;
        const int cp = r - t * Cgp;
        const int bu = t / kwp;
        const int bv = t - bu * kwp;
        const int f = cp / Cg;
        const int c = cp - f * Cg;
        const int fu = f / S;
        const int u = S * bu + fu;
        const int v = S * bv + f - fu * S;
        bf16_t x = 0;
        if (f < S * S && u < kh && v < kw)
            x = W[(((long)o * Cg + c) * kh + u) * kw + v];
        Wp[e] = x;
    }
}

// Phase-stacked data-gradient weights (as dgrad_weight_transform_kernel) with
// the reduction index tap-major over padded channels:
// Wt[g][m = (c, fh, fw)][(th*Tw + tw)*Kgp + k] = W[g*Kg + k][c][fh + sh*(Th-1-th)][fw + sw*(Tw-1-tw)],
// zero past the kernel edge, for k >= Kg and for r >= Th*Tw*Kgp (rows padded to Rtp).
__global__ void __launch_bounds__(256)
dgrad_weights_bf16_kernel(const bf16_t* __restrict__ W, bf16_t* __restrict__ Wt, int G, int Kg,
                          int Kgp, int Cg, int kh, int kw, int sh, int sw, int Th, int Tw, int Rtp,
                          int blocked)
{
    const int Mt = Cg * sh * sw;
    const long total = (long)G * Mt * Rtp;
    for (long e = blockIdx.x * (long)blockDim.x + threadIdx.x; e < total;
         e += (long)gridDim.x * blockDim.x) {
        const int r = (int)(e % Rtp);
        const long gm = e / Rtp;
        const int m = (int)(gm % Mt);
        const int g = (int)(gm / Mt);
        int t, k;
        if (blocked) {  // ((k / 64)*Th*Tw + t)*64 + k % 64
            const int b = r / (Th * Tw * 64);
            const int rem = r - b * Th * Tw * 64;
            t = rem >> 6;
            k = b * 64 + (rem & 63);
        } else {
            t = r / Kgp;
            k = r - t * Kgp;
        }
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

template <int MT, int WM, int WN, int MI, int NI, int NS, int EPI, int MASK>
hipError_t launch_gemm(const GemmBf16Params& p, hipStream_t s)
{
    constexpr int TM = WM * MI * MT, TN = WN * NI * MT;
    const int64_t tiles = (int64_t)((p.Ncol + TN - 1) / TN) * ((p.M + TM - 1) / TM) * p.G;
    const int64_t per_xcd = (tiles + 7) / 8;
    hipLaunchKernelGGL((conv_gemm_bf16_kernel<MT, WM, WN, MI, NI, NS, EPI, MASK>),
                       dim3((unsigned)(per_xcd * 8)), dim3(64 * WM * WN), 0, s, p);
    return hipGetLastError();
}

template <int NS, int EPI, int MASK>
hipError_t launch_gemm_tile(const GemmBf16Params& p, int tile, hipStream_t s)
{
    switch (tile) {
    case BTILE_128x256:
        return launch_gemm<32, 2, 4, 2, 2, NS, EPI, MASK>(p, s);
    case BTILE_96x256:
        return launch_gemm<32, 1, 8, 3, 1, NS, EPI, MASK>(p, s);
    case BTILE_64x256:
        return launch_gemm<32, 1, 4, 2, 2, NS, EPI, MASK>(p, s);
    case BTILE_48x256:
        return launch_gemm<16, 1, 8, 3, 2, NS, EPI, MASK>(p, s);
    default:
        return hipErrorInvalidValue;
    }
}

template <int EPI, int MASK>
hipError_t launch_gemm_pipe(const GemmBf16Params& p, int tile, int pipe, hipStream_t s)
{
    switch (pipe) {
    case BPIPE_2:
        return launch_gemm_tile<2, EPI, MASK>(p, tile, s);
    case BPIPE_3:
        return launch_gemm_tile<3, EPI, MASK>(p, tile, s);
    default:
        return hipErrorInvalidValue;
    }
}

// epi 2: the tiles of 32-row blocks with four waves of 64 columns
template <int MASK>
hipError_t launch_stage_below(const GemmBf16Params& p, int tile, int pipe, hipStream_t s)
{
    const bool three = pipe == BPIPE_3;
    switch (tile) {
    case BTILE_128x256:
        return three ? launch_gemm<32, 2, 4, 2, 2, 3, 2, MASK>(p, s)
                     : launch_gemm<32, 2, 4, 2, 2, 2, 2, MASK>(p, s);
    case BTILE_64x256:
        return three ? launch_gemm<32, 1, 4, 2, 2, 3, 2, MASK>(p, s)
                     : launch_gemm<32, 1, 4, 2, 2, 2, 2, MASK>(p, s);
    default:
        return hipErrorInvalidValue;
    }
}

template <int WM, int WN, int MI, int NI>
hipError_t launch_wg(const WgradBf16Params& p, hipStream_t s)
{
    constexpr int TM = WM * MI * 32, TN = WN * NI * 32;
    const int64_t per_unit = (int64_t)((p.Rw + TN - 1) / TN) * ((p.Kg + TM - 1) / TM);
    const int64_t units = (int64_t)p.G * p.splits;
    // unit order: whole rounds of 8 units (the blocks past the last unit exit)
    const int64_t tiles = p.unit_order ? (units + 7) / 8 * 8 * per_unit : units * per_unit;
    if (tiles > INT_MAX)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL((conv_wgrad_bf16_kernel<WM, WN, MI, NI, 3>), dim3((unsigned)tiles),
                       dim3(64 * WM * WN), 0, s, p);
    return hipGetLastError();
}

}  // namespace

int bf16_tile_m(int tile)
{
    switch (tile) {
    case BTILE_128x256:
        return 128;
    case BTILE_96x256:
        return 96;
    case BTILE_64x256:
        return 64;
    case BTILE_48x256:
        return 48;
    default:
        return 0;
    }
}

hipError_t launch_conv_gemm_bf16(const GemmBf16Params& p, int epi, int tile, int pipe,
                                 hipStream_t s)
{
    if (p.Ncol == 0)
        return hipSuccess;
    const bool wide = p.Cgp % 8 == 0 && p.Ctot % 8 == 0 && p.Cg8 * 8 == p.Cgp && p.vstr == p.Ctot;
    const bool narrow = (p.Cgp == 1 || p.Cgp == 2 || p.Cgp == 4) && p.Ctot == p.Cgp && p.G == 1 &&
                        p.Cg8 == 1 && p.vstr == 8;
    if (p.Rp % kBf16TK != 0 || !(wide || narrow) || p.KC * 8 > p.Rp ||
        p.KC != p.kh * p.kw * p.Cg8)
        return hipErrorInvalidValue;
    if (epi == 0)
        return launch_gemm_pipe<0, 0>(p, tile, pipe, s);
    if (epi == 2) {
        // stride 1, the column grid the image itself, whole quads of rows
        if (p.psh != 1 || p.psw != 1 || p.OH != p.OutH || p.OW != p.OutW ||
            p.a0h != p.oph || p.a0w != p.opw || p.M != p.Cg_out || p.M % 4 != 0 ||
            p.Cg_out % 4 != 0 || p.s_Ktot % 4 != 0 || !p.Sh || !p.Ssum ||
            p.s_T < stage_below_terms(p.Ncol) || p.s_tb < 0 || p.s_lb < 0 ||
            p.s_Hp < p.s_tb + p.OutH || p.s_Wp < p.s_lb + p.OutW ||
            (int64_t)p.G * p.Cg_out > p.s_Ktot ||
            (int64_t)p.N * p.s_Hp * p.s_Wp * p.s_Ktot * 2 > (int64_t)p.Sh_bytes ||
            (int64_t)p.G * p.Cg_out * p.s_T * 4 > (int64_t)p.Ssum_bytes)
            return hipErrorInvalidValue;
        if (!p.Omask)
            return launch_stage_below<0>(p, tile, pipe, s);
        return p.omask_f32 ? launch_stage_below<2>(p, tile, pipe, s)
                           : launch_stage_below<1>(p, tile, pipe, s);
    }
    if (!p.Omask)
        return launch_gemm_pipe<1, 0>(p, tile, pipe, s);
    return p.omask_f32 ? launch_gemm_pipe<1, 2>(p, tile, pipe, s)
                       : launch_gemm_pipe<1, 1>(p, tile, pipe, s);
}

int stage_below_terms(int64_t ncol) { return (int)(4 * ((ncol + 255) / 256)); }

int bf16_wgrad_tile_m(int tile) { return tile == BWTILE_96x256 ? 96 : 128; }

hipError_t launch_conv_wgrad_bf16(const WgradBf16Params& p, int tile, hipStream_t s)
{
    const bool narrow = (p.Cgp == 1 || p.Cgp == 2 || p.Cgp == 4) && p.Ctot == p.Cgp && p.G == 1;
    if ((p.Cgp % 8 != 0 && !narrow) || p.Kgp % 8 != 0 || p.cols_per_split % kBf16WgradTK != 0)
        return hipErrorInvalidValue;
    switch (tile) {
    case BWTILE_128x256:
        return launch_wg<2, 4, 2, 2>(p, s);
    case BWTILE_96x256:
        return launch_wg<1, 8, 3, 1>(p, s);
    default:
        return hipErrorInvalidValue;
    }
}

hipError_t launch_wgrad_reduce_perm(const float* P, float* dW, int K, int Rw, int Cgp, int Cg,
                                    int kh, int kw, int kwp, int S, int splits, int accumulate,
                                    hipStream_t s)
{
    const int count = K * Rw;
    if (count == 0)
        return hipSuccess;
    hipLaunchKernelGGL(wgrad_reduce_perm_kernel, dim3((count + kPermCols - 1) / kPermCols),
                       dim3(kPermParts * kPermCols), 0, s, P, dW, K, Rw, Cgp, Cg, kh, kw, kwp, S,
                       splits, accumulate);
    return hipGetLastError();
}

template <typename T>
hipError_t launch_stage(const T* X, uint16_t* Xp, int N, int C, int H, int W, int Cg, int Cgp,
                        int Ctot, int Hp, int Wp, int tb, int lb, hipStream_t s)
{
    if (Ctot < 8) {  // one group of 1, 2 or 4 channels
        // (the channel offsets stay below 2^32 bytes, range-checked)
        if ((int64_t)Ctot * H * W * (int64_t)sizeof(T) >= (int64_t(1) << 32))
            return hipErrorInvalidValue;
        const int per_image = Hp * Wp * Ctot / 8;
        const FastDiv dwp = make_fastdiv((uint32_t)Wp);
        // (images in launches of at most 65535: the grid's y extent)
        for (int n0 = 0; n0 < N; n0 += 65535) {
            const dim3 grid((unsigned)((per_image + 255) / 256), (unsigned)std::min(N - n0, 65535));
            const T* Xn = X + (size_t)n0 * Cg * H * W;
            uint16_t* Xpn = Xp + (size_t)n0 * per_image * 8;
            if (Ctot == 4)
                hipLaunchKernelGGL((stage_narrow_bf16_kernel<4, T>), grid, dim3(256), 0, s, Xn,
                                   Xpn, Cg, H, W, Hp, Wp, tb, lb, dwp);
            else if (Ctot == 2)
                hipLaunchKernelGGL((stage_narrow_bf16_kernel<2, T>), grid, dim3(256), 0, s, Xn,
                                   Xpn, Cg, H, W, Hp, Wp, tb, lb, dwp);
            else
                hipLaunchKernelGGL((stage_narrow_bf16_kernel<1, T>), grid, dim3(256), 0, s, Xn,
                                   Xpn, Cg, H, W, Hp, Wp, tb, lb, dwp);
        }
        return hipGetLastError();
    }
    // (the channel offsets, up to one tile past the last channel, stay below
    // 2^32 bytes: range-checked, never wrapped)
    const bool offsets_fit = ((int64_t)C + kStageRowCh) * H * W * (int64_t)sizeof(T) <
                             (int64_t(1) << 32);
    if (W <= kStageRowPixels && Ctot >= 32 && Cgp == Cg && offsets_fit) {
        const int RH = kStageRowPixels / W;
        const int rchunks = (Hp + RH - 1) / RH;
        const int ctiles = (Ctot + kStageRowCh - 1) / kStageRowCh;
        hipLaunchKernelGGL((stage_rows_bf16_kernel<T>),
                           dim3((unsigned)((int64_t)N * rchunks * ctiles)), dim3(256), 0, s, X, Xp,
                           C, H, W, Cg, Cgp, Ctot, Hp, Wp, tb, lb, RH, rchunks, ctiles);
        return hipGetLastError();
    }
    const int ct = Ctot <= 8 ? 8 : Ctot <= 16 ? 16 : Ctot <= 32 ? 32 : 64;
    const int pt = ct == 8 ? stage_tile_pixels<8>() : ct == 16 ? stage_tile_pixels<16>()
                 : ct == 32 ? stage_tile_pixels<32>() : stage_tile_pixels<64>();
    const int ptiles = (Hp * Wp + pt - 1) / pt;
    const int ctiles = (Ctot + ct - 1) / ct;
    const dim3 grid((unsigned)((int64_t)ptiles * ctiles * N));
#define CAFFE_STAGE_LAUNCH(CT)                                                                    \
    hipLaunchKernelGGL((stage_nhwc_bf16_kernel<CT, T>), grid, dim3(256), 0, s, X, Xp, C, H, W, Cg, \
                       Cgp, Ctot, Hp, Wp, tb, lb, ptiles, ctiles)
    switch (ct) {
    case 8:
        CAFFE_STAGE_LAUNCH(8);
        break;
    case 16:
        CAFFE_STAGE_LAUNCH(16);
        break;
    case 32:
        CAFFE_STAGE_LAUNCH(32);
        break;
    default:
        CAFFE_STAGE_LAUNCH(64);
        break;
    }
#undef CAFFE_STAGE_LAUNCH
    return hipGetLastError();
}

hipError_t launch_stage_nhwc_bf16(const void* X, int x_f32, uint16_t* Xp, int N, int C, int H,
                                  int W, int Cg, int Cgp, int Ctot, int Hp, int Wp, int tb, int lb,
                                  hipStream_t s)
{
    if (N == 0)
        return hipSuccess;
    if (x_f32)
        return launch_stage((const float*)X, Xp, N, C, H, W, Cg, Cgp, Ctot, Hp, Wp, tb, lb, s);
    return launch_stage((const uint16_t*)X, Xp, N, C, H, W, Cg, Cgp, Ctot, Hp, Wp, tb, lb, s);
}

int diff_prep_terms(int N, int HWp)
{
    return N * std::max(1, (HWp + kDiffPrepPixels - 1) / kDiffPrepPixels);
}

hipError_t launch_diff_prep_bf16(const float* G, const float* Y, uint16_t* Dh, float* sums, int N,
                                 int K, int H, int W, int Kg, int Kgp, int Ktot, int Hp, int Wp,
                                 int tb, int lb, int relu, hipStream_t s)
{
    if (N == 0)
        return hipSuccess;
    const int ctiles = (Ktot + 63) / 64;
    const int runs = diff_prep_terms(N, Hp * Wp) / N;
    const dim3 grid((unsigned)((int64_t)ctiles * N * runs));
    if (relu)
        hipLaunchKernelGGL(diff_prep_bf16_kernel<true>, grid, dim3(256), 0, s, G, Y, Dh, sums, N,
                           K, H, W, Kg, Kgp, Ktot, Hp, Wp, tb, lb, ctiles, runs);
    else
        hipLaunchKernelGGL(diff_prep_bf16_kernel<false>, grid, dim3(256), 0, s, G, Y, Dh, sums, N,
                           K, H, W, Kg, Kgp, Ktot, Hp, Wp, tb, lb, ctiles, runs);
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
                                    int kh, int kw, int kwp, int S, int Rp, hipStream_t s)
{
    const long total = (long)K * Rp;
    if (total == 0)
        return hipSuccess;
    hipLaunchKernelGGL(pack_weights_bf16_kernel, dim3(grid_1d(total)), dim3(256), 0, s, W, Wp, K,
                       Cg, Cgp, kh, kw, kwp, S, Rp);
    return hipGetLastError();
}

// Space-to-depth staging by S (a strided layer as a stride-1 one):
// Xp[n][a][b][(fu*S + fv)*C + c] = X[n][c][S*a + fu - ph][S*b + fv - pw] (0
// outside the image and for channels past C*S*S, up to Csp).  One block per
// (RA staged rows, image n): the S*RA source rows of every channel go to LDS
// with lanes along the row (coalesced, eight loads in flight per thread),
// then each thread writes 16-byte chunks of 8 staged channels, lanes along
// (pixel, chunk).
template <typename T>
__global__ void __launch_bounds__(256)
stage_s2d_bf16_kernel(const T* __restrict__ X, bf16_t* __restrict__ Xp, int C, int H, int W,
                      int S, int ph, int pw, int XHp, int XWp, int Csp, int RA, FastDiv div_c8,
                      FastDiv div_xwp)
{
    extern __shared__ bf16_t srows[];  // [C][S * RA][XWp * S]
    __shared__ int ctab[64];           // staged channel -> its (c, fu) row and fv in srows
    const int tid = threadIdx.x;
    const int a0 = blockIdx.x * RA;
    const int na = min(RA, XHp - a0);
    const int n = blockIdx.y;
    const int RW = XWp * S;
    const int SR = S * RA;              // source rows per channel
    const int Cs = C * S * S;
    if (tid < Csp) {
        int t = -1;
        if (tid < Cs) {
            const int f = tid / C;
            const int c = tid - f * C;
            const int fu = f / S;
            t = (c * SR + fu) * RW + (f - fu * S);
        }
        ctab[tid] = t;
    }
    const uint32_t plane = (uint32_t)(H * W) * (uint32_t)sizeof(T);
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(X + (size_t)n * C * H * W, (uint32_t)C * plane);
    // source rows rr = c * SR + r, eight at a time, lanes along the row
    const int nrows = C * SR;
    for (int rr0 = 0; rr0 < nrows; rr0 += 8) {
        for (int x = tid; x < RW; x += 256) {
            const int w = x - pw;
            const bool win = (unsigned)w < (unsigned)W;
            T v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int rr = rr0 + u;  // (uniform)
                const int c = rr / SR;
                const int h = S * a0 + (rr - c * SR) - ph;
                const bool in = rr < nrows && win && (unsigned)h < (unsigned)H;
                const uint32_t voff =
                    in ? (uint32_t)c * plane + (uint32_t)(h * W + w) * (uint32_t)sizeof(T) : kOob;
                v[u] = load_elem<T>(rx, voff, 0u);
            }
#pragma unroll
            for (int u = 0; u < 8; ++u)
                if (rr0 + u < nrows)
                    srows[(rr0 + u) * RW + x] = to_bf16(v[u]);
        }
    }
    __syncthreads();
    // 16-byte chunks of 8 staged channels, lanes along (pixel, chunk)
    const int C8 = Csp / 8;
    for (int id = tid; id < na * XWp * C8; id += 256) {
        const int pl = (int)fdiv((uint32_t)id, div_c8);  // (row of the block, b)
        const int q = id - pl * C8;
        const int ra = (int)fdiv((uint32_t)pl, div_xwp);
        const int b = pl - ra * XWp;
        const int base = S * (ra * RW + b);
        uint32_t wv[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int t0 = ctab[8 * q + 2 * k], t1 = ctab[8 * q + 2 * k + 1];
            const uint32_t lo = t0 >= 0 ? srows[t0 + base] : 0u;
            const uint32_t hi = t1 >= 0 ? srows[t1 + base] : 0u;
            wv[k] = lo | (hi << 16);
        }
        *(u32x4*)&Xp[(((size_t)n * XHp + a0 + ra) * XWp + b) * Csp + 8 * q] =
            u32x4{wv[0], wv[1], wv[2], wv[3]};
    }
}

hipError_t launch_stage_s2d_bf16(const void* X, int x_f32, uint16_t* Xp, int N, int C, int H,
                                 int W, int S, int ph, int pw, int XHp, int XWp, int Csp,
                                 hipStream_t s)
{
    if (N == 0)
        return hipSuccess;
    // staged rows per block: at most 16 KB of source rows in LDS (eight
    // blocks per compute unit, so that one block's loads overlap another's
    // stores)
    const size_t row_lds = (size_t)C * S * XWp * S * 2;
    if (row_lds > 64 * 1024 || Csp % 8 != 0 || C * S * S > Csp || Csp > 64 || N > 65535 ||
        (int64_t)C * H * W * 4 >= (int64_t(1) << 31))
        return hipErrorInvalidValue;
    const int RA = (int)std::max<size_t>(1, std::min<size_t>(8, (16 * 1024) / row_lds));
    const dim3 grid((unsigned)((XHp + RA - 1) / RA), (unsigned)N);
    const size_t lds = row_lds * RA;
    const FastDiv dc8 = make_fastdiv((uint32_t)(Csp / 8)), dxw = make_fastdiv((uint32_t)XWp);
    if (x_f32)
        hipLaunchKernelGGL(stage_s2d_bf16_kernel<float>, grid, dim3(256), lds, s,
                           (const float*)X, Xp, C, H, W, S, ph, pw, XHp, XWp, Csp, RA, dc8, dxw);
    else
        hipLaunchKernelGGL(stage_s2d_bf16_kernel<bf16_t>, grid, dim3(256), lds, s,
                           (const bf16_t*)X, Xp, C, H, W, S, ph, pw, XHp, XWp, Csp, RA, dc8, dxw);
    return hipGetLastError();
}

hipError_t launch_dgrad_weights_bf16(const uint16_t* W, uint16_t* Wt, int G, int Kg, int Kgp,
                                     int Cg, int kh, int kw, int sh, int sw, int Th, int Tw,
                                     int Rtp, int blocked, hipStream_t s)
{
    const long total = (long)G * Cg * sh * sw * Rtp;
    if (total == 0)
        return hipSuccess;
    if (blocked && Kgp % 64 != 0)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(dgrad_weights_bf16_kernel, dim3(grid_1d(total)), dim3(256), 0, s, W, Wt, G,
                       Kg, Kgp, Cg, kh, kw, sh, sw, Th, Tw, Rtp, blocked);
    return hipGetLastError();
}

}  // namespace caffe_hip
