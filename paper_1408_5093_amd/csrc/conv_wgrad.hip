// conv_wgrad.hip -- weight gradient of the convolution layer (the "gradients
// with respect to the parameters" of the paper's Sec. 3.2 backward pass) as a
// split-K implicit GEMM on gfx950 fp32 MFMA.
//
// Per group g:  dW_g[m][r] = sum_col D[n][g*Kg + m][i][j] * X[n][g*Cg + c][i*sh - ph + u][j*sw - pw + v]
//   m   over Kg (output channels of the group)        -> GEMM rows, TM per workgroup
//   r   = (c, u, v) over Cg x kh x kw                   -> GEMM columns, TN per workgroup
//   col = (n, i, j) over N x OH x OW                    -> reduction, split into `splits`
//                                                        contiguous ranges, TK per stage
// Each (tile, split) writes its own partial sum; a separate kernel adds the
// partials in a fixed order, so the result is reproducible bit for bit.
//
// Both operands are gathered with lanes running along the reduction index
// (consecutive output pixels), which keeps the HBM/L2 reads coalesced.
#include "device_common.h"
#include "kernels.h"

namespace caffe_hip {

// The logical tile of this workgroup (workgroup L runs on XCD L % 8):
// linear; XCD-contiguous (tile (L % 8) * per_xcd + L / 8, per_xcd = the
// grid / 8); or unit order, where slot s = L / 8 of XCD x takes tile s % U of
// unit (s / U) * 8 + x, U = per_unit the tiles of one (group, split) unit.
__device__ __forceinline__ int wgrad_tile_index(const WgradParams& p, int per_unit)
{
    if (p.unit_order) {
        const int slot = blockIdx.x >> 3;
        return ((slot / per_unit) * 8 + (blockIdx.x & 7)) * per_unit + slot % per_unit;
    }
    const int per_xcd = gridDim.x >> 3;
    return p.xcd_order ? (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3) : blockIdx.x;
}

// Workgroups of a weight-gradient launch: whole rounds of 8 XCDs of tiles,
// or of units in unit order (the workgroups past the last tile exit).
static int64_t wgrad_grid(const WgradParams& p, int64_t per_unit)
{
    const int64_t units = (int64_t)p.G * p.splits;
    return p.unit_order ? (units + 7) / 8 * 8 * per_unit : (units * per_unit + 7) / 8 * 8;
}

template <int WM, int WN, int MI, int NI, int TK, int KH, int KW, int SH, int SW>
__global__ void __launch_bounds__(64 * WM * WN)
conv_wgrad_f32_kernel(const WgradParams p)
{
    constexpr int MT = 32;
    constexpr int NT = 64 * WM * WN;
    constexpr int TM = WM * MI * MT;
    constexpr int TN = WN * NI * MT;
    constexpr int RS = NT / TK;       // rows covered by one pass of the block
    constexpr int EA = TM / RS;       // A elements per thread per stage
    constexpr int EB = TN / RS;       // B elements per thread per stage
    static_assert(NT % TK == 0 && TM % RS == 0 && TN % RS == 0, "wgrad mapping");
    static_assert(TK % 2 == 0, "stage depth");

    // Row stride = 2 (mod 32) keeps the lane-along-k LDS writes conflict-free.
    __shared__ float As[2][TK][TM + 2];
    __shared__ float Bs[2][TK][TN + 2];

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
    // Tap tiles vary fastest, then row tiles (see wgrad_tile_index): in the
    // XCD-contiguous and unit orders the workgroups sharing a split's diff
    // rows run together on one XCD.
    const int n_rt = (p.R + TN - 1) / TN;
    const int n_mt = (p.Kg + TM - 1) / TM;
    const int T = wgrad_tile_index(p, n_rt * n_mt);
    if (T >= n_rt * n_mt * p.G * p.splits)
        return;
    const int rt = T % n_rt;
    const int mt = (T / n_rt) % n_mt;
    const int g = (T / (n_rt * n_mt)) % p.G;
    const int split = T / (n_rt * n_mt * p.G);
    const int m0 = mt * TM;
    const int r0 = rt * TN;
    const int IH = p.IH, IW = p.IW, IHW = IH * IW;
    const int OHW = p.OH * p.OW;

    const int col_begin = split * p.cols_per_split;
    const int col_end = min(p.Ncol, col_begin + p.cols_per_split);

    const __amdgpu_buffer_rsrc_t rd = make_rsrc(p.D, p.D_bytes);

    const __amdgpu_buffer_rsrc_t rx = make_rsrc(p.X, p.X_bytes);

    const int kc = tid % TK;  // reduction index within a stage
    const int rw = tid / TK;  // row within one pass

    // Per-thread A rows (output channels) and B rows (taps), fixed for the
    // kernel.  Neither needs a row mask: A rows past Kg and B rows past R only
    // feed accumulator rows / columns that the epilogue never stores, and
    // their loads stay inside the tensors or read 0.  A columns need none
    // either: splits are whole stages, so the only columns past a split's end
    // lie past Ncol, in images n >= N, which are outside D (read as 0).
    const int a_off0 = (g * p.Kg + m0 + rw) * OHW;
    // Per-thread tap table.  MASKED (a compile-time kernel with kh*kw < 32):
    // entry q packs the byte offset (c*IH*IW + u*IW + v) * 4 in bits 5..31 and
    // the tap index u*kw + v in bits 0..4, and the bounds test reads the tap's
    // bit of the column's in-image mask.  Otherwise, with a compile-time
    // kernel (PACK): offset c*IH*IW + u*IW + v in bits 0..21, u in 22..26, v
    // in 27..31 (the launcher checks Cg*IH*IW < 2^22 and kh, kw <= 32), taps
    // past R flagged in r_bad.
    constexpr bool PACK = KH != 0;
    constexpr bool MASKED = KH != 0 && KH * KW < 32;
    constexpr uint32_t kRep = [] {
        uint32_t r = 0;
        for (int u = 0; u < (MASKED ? KH : 0); ++u)
            r |= 1u << (u * KW);
        return r;
    }();
    int b_off[EB];
    int b_uv[PACK ? 1 : EB];
    uint32_t r_bad = 0;
#pragma unroll
    for (int q = 0; q < EB; ++q) {
        const int r = r0 + rw + RS * q;
        const int rr_ = r < p.R ? r : 0;
        const int c = rr_ / khw;
        const int rr = rr_ - c * khw;
        const int u = rr / kw;
        const int v = rr - u * kw;
        if (r >= p.R)
            r_bad |= 1u << q;
        if constexpr (MASKED) {
            b_off[q] = (int)((uint32_t)((c * IHW + u * IW + v) * 4) << 5 | (uint32_t)(u * KW + v));
        } else if constexpr (PACK) {
            b_off[q] = (c * IHW + u * IW + v) | (u << 22) | (v << 27);
        } else {
            b_off[q] = c * IHW + u * IW + v;
            b_uv[q] = u | (v << 16);
        }
    }

    float rA[EA], rB[EB];
    // bias-gradient partials: in the first tap tile's workgroups, thread t < TM
    // owns row t and adds the staged (masked) diff of its row, stage by stage
    const bool want_db = p.dbp != nullptr && rt == 0;
    float dsum = 0.f;

    auto load_stage = [&](int cbase) {
        // The tap table is decoded afresh each stage: the empty asm hides its
        // loop invariance, which would otherwise keep decoded copies live in
        // extra registers for the whole loop.
#pragma unroll
        for (int q = 0; q < EB; ++q)
            asm volatile("" : "+v"(b_off[q]));
        const int col = cbase + kc;
        const int n = (int)fdiv((uint32_t)col, p.div_ohw);
        const int pix = col - n * OHW;
        const int i = (int)fdiv((uint32_t)pix, p.div_ow);
        const int j = pix - i * p.OW;
        uint32_t dbase4 = (uint32_t)(n * p.K * OHW + pix + a_off0) * 4u;
        // materialised once, so each row below is one add (left alone, the
        // compiler re-derives every row's offset with a 64-bit multiply-add)
        asm volatile("" : "+v"(dbase4));
        const int ih0 = i * sh - p.ph;
        const int iw0 = j * sw - p.pw;
        const int xbase = (n * p.C + g * p.Cg) * IHW + ih0 * IW + iw0;
#pragma unroll
        for (int q = 0; q < EA; ++q)
            rA[q] = buf_ld_f32(rd, dbase4 + (uint32_t)(RS * q * OHW) * 4u);
        if constexpr (MASKED) {
            // taps of this column's window that lie in the image, bit u*KW + v
            // (none for a column past Ncol)
            const int ulo = min(max(-ih0, 0), KH), uhi = max(min(IH - ih0, KH), ulo);
            const int vlo = min(max(-iw0, 0), KW), vhi = max(min(IW - iw0, KW), vlo);
            const uint32_t wbits = (1u << vhi) - (1u << vlo);
            const uint32_t rows = (1u << (uhi * KW)) - (1u << (ulo * KW));
            const uint32_t nok = col < p.Ncol ? ~(wbits * kRep & rows) : ~0u;
            const uint32_t xb4 = (uint32_t)xbase * 4u;
#pragma unroll
            for (int q = 0; q < EB; ++q) {
                const uint32_t e = (uint32_t)b_off[q];
                rB[q] = buf_ld_f32(rx, (xb4 + (e >> 5)) | (((nok >> (e & 31u)) & 1u) << 31));
            }
        } else if (PACK && __all(ih0 >= 0 && ih0 + kh <= IH && iw0 >= 0 && iw0 + kw <= IW)) {
            // every column of the wave has its whole window inside the image
            // (every wave of an unpadded layer): no per-tap bounds test.  A
            // column past Ncol lies in an image n >= N, outside X (reads 0);
            // taps past R only feed columns that are never stored.
#pragma unroll
            for (int q = 0; q < EB; ++q)
                rB[q] = buf_ld_f32(rx, (uint32_t)(xbase + (b_off[q] & 0x3fffff)) * 4u);
        } else {
            const uint32_t cbad = (uint32_t)(col >= col_end) << 31;
#pragma unroll
            for (int q = 0; q < EB; ++q) {
                int ih, iw, boff;
                if constexpr (PACK) {
                    ih = ih0 + ((b_off[q] >> 22) & 31);
                    iw = iw0 + ((uint32_t)b_off[q] >> 27);
                    boff = b_off[q] & 0x3fffff;
                } else {
                    ih = ih0 + (b_uv[q] & 0xffff);
                    iw = iw0 + (b_uv[q] >> 16);
                    boff = b_off[q];
                }
                const uint32_t bad = ((uint32_t)((unsigned)ih >= (unsigned)IH) |
                                      (uint32_t)((unsigned)iw >= (unsigned)IW)) << 31;
                const uint32_t off = ((uint32_t)(xbase + boff) * 4u) | cbad | bad |
                                     (((r_bad >> q) & 1u) << 31);
                rB[q] = buf_ld_f32(rx, off);
            }
        }
    };

    auto store_stage = [&](int buf) {
#pragma unroll
        for (int q = 0; q < EA; ++q)
            As[buf][kc][rw + RS * q] = rA[q];
#pragma unroll
        for (int q = 0; q < EB; ++q)
            Bs[buf][kc][rw + RS * q] = rB[q];
    };

    floatx16 acc[MI][NI];
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int ni = 0; ni < NI; ++ni)
            acc[mi][ni] = floatx16{};

    const int nst = col_end > col_begin ? (col_end - col_begin + TK - 1) / TK : 0;
    if (nst > 0) {
        load_stage(col_begin);
        store_stage(0);
    }
    __syncthreads();

    const int arow = wm * MI * MT + (lane & 31);
    const int bcol = wn * NI * MT + (lane & 31);
    const int kl = lane >> 5;

    for (int s = 0; s < nst; ++s) {
        const int cur = s & 1;
        if (s + 1 < nst)
            load_stage(col_begin + (s + 1) * TK);
        if (want_db && tid < TM) {
#pragma unroll
            for (int k = 0; k < TK; ++k)
                dsum += As[cur][k][tid];
        }
        // rolling fragment prefetch, as in the forward kernel
        constexpr int KS = TK / 2;
        constexpr int PF = 2;
        float fa[PF + 1][MI], fb[PF + 1][NI];
        auto read_frag = [&](int ks, int slot) {
#pragma unroll
            for (int mi = 0; mi < MI; ++mi)
                fa[slot][mi] = As[cur][2 * ks + kl][arow + mi * MT];
#pragma unroll
            for (int ni = 0; ni < NI; ++ni)
                fb[slot][ni] = Bs[cur][2 * ks + kl][bcol + ni * MT];
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
                    acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x2f32(
                        fa[ks % (PF + 1)][mi], fb[ks % (PF + 1)][ni], acc[mi][ni], 0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
        }
        if (s + 1 < nst)
            store_stage(cur ^ 1);
        __syncthreads();
    }

    if (want_db) {
        const int m = m0 + tid;
        if (tid < TM && m < p.Kg)
            p.dbp[split * p.K + g * p.Kg + m] = dsum;
    }

    // Partial result P[split][g*Kg + m][r]: lanes run along r (contiguous).
    const __amdgpu_buffer_rsrc_t rp = make_rsrc(p.P, p.P_bytes);
    const int pbase = split * p.K * p.R;
#pragma unroll
    for (int ni = 0; ni < NI; ++ni) {
        const int r = r0 + bcol + ni * MT;
#pragma unroll
        for (int mi = 0; mi < MI; ++mi) {
#pragma unroll
            for (int q = 0; q < 16; ++q) {
                const int m = m0 + wm * MI * MT + mi * MT + 8 * (q >> 2) + 4 * (lane >> 5) + (q & 3);
                const bool ok = m < p.Kg && r < p.R;
                const uint32_t off = ok ? (uint32_t)(pbase + (g * p.Kg + m) * p.R + r) * 4u : kOob;
                buf_st_f32(acc[mi][ni][q], rp, off);
            }
        }
    }
}

// ------------------------------------------------------------ quad order
// Layers with Cg % 4 == 0 and a kernel of kh*kw < 32 taps run the same
// split-K GEMM with its tap dimension in the order
//   r' = ((c / 4) * kh*kw + u*kw + v) * 4 + c % 4
// (four channels of one tap side by side).  A thread's loader rows are
// r' = r0 + rw + 16 q with rw = 4 * wave + lane / 16, so c % 4 is the lane's
// (a fixed channel-plane offset) and r' / 4 = r0 / 4 + wave + 4 q is
// wave-uniform: each B load takes the column's window base in the lane
// offset and the tap's offset in the scalar offset, and its bounds test is
// one bit of the column's tap mask.  A rows m0 + rw + 16 q split the same
// way.  The columns' bases and masks come from a table written once per call
// (wgrad_col_table_kernel), so a stage decodes no pixel indices.  The
// epilogue maps r' back to r = c*kh*kw + u*kw + v.
//
// LDS tiles hold each wave's MFMA row blocks interleaved in pairs
// (position 2*(m % 32) + block parity), so one 8-byte read fetches the
// fragments of two blocks at an immediate offset.

// Position of tile row m = 32 * sub + l within its LDS row, for a tile whose
// waves own slabs of NSUB 32-row blocks.
template <int NSUB>
__device__ __forceinline__ int quad_lds_pos(int sub, int l)
{
    const int slab = sub / NSUB, mi = sub % NSUB;
    const bool pair = (mi | 1) < NSUB;
    return slab * NSUB * 32 + (mi / 2) * 64 + (pair ? 2 * l + (mi & 1) : l);
}

template <int WM, int WN, int MI, int NI, int KH, int KW>
__global__ void __launch_bounds__(64 * WM * WN) __attribute__((amdgpu_waves_per_eu(4)))
conv_wgrad_quad_f32_kernel(const WgradParams p)
{
    constexpr int MT = 32;
    constexpr int NT = 64 * WM * WN;
    constexpr int TM = WM * MI * MT;
    constexpr int TN = WN * NI * MT;
    constexpr int TK = 16;
    constexpr int RS = NT / TK;  // loader rows per pass
    constexpr int EA = TM / RS;  // A elements per thread per stage
    constexpr int EB = TN / RS;  // B elements per thread per stage
    constexpr int KHW = KH * KW;
    static_assert(RS == 16 && TM % 32 == 0 && TN % 32 == 0, "quad loader mapping");
    static_assert(KHW < 32, "one mask bit per tap");

    // rows of 8-byte aligned length; the stride (2 mod 32 words) keeps the
    // loader's 8-byte writes conflict-free
    __shared__ float As[2][TK][TM + 2];
    __shared__ float Bs[2][TK][TN + 2];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave % WM;
    const int wn = wave / WM;
    const int n_rt = (p.R + TN - 1) / TN;
    const int n_mt = (p.Kg + TM - 1) / TM;
    const int T = wgrad_tile_index(p, n_rt * n_mt);
    if (T >= n_rt * n_mt * p.G * p.splits)
        return;
    const int rt = T % n_rt;
    const int mt = (T / n_rt) % n_mt;
    const int g = (T / (n_rt * n_mt)) % p.G;
    const int split = T / (n_rt * n_mt * p.G);
    const int m0 = mt * TM;
    const int r0 = rt * TN;
    const int IW = p.IW, IHW = p.IH * p.IW;
    const int OHW = p.OH * p.OW;
    const int col_begin = split * p.cols_per_split;
    const int col_end = min(p.Ncol, col_begin + p.cols_per_split);

    const __amdgpu_buffer_rsrc_t rd = make_rsrc(p.D, p.D_bytes);
    // X through a base p.xpad elements early: every window base in the table
    // is then >= 0 and every tap offset below is >= 0
    const __amdgpu_buffer_rsrc_t rx =
        make_rsrc((const char*)p.X - 4 * (size_t)p.xpad, p.X_bytes + 4u * (uint32_t)p.xpad);
    const __amdgpu_buffer_rsrc_t rtab = make_rsrc(p.T, p.T_bytes);

    const int kc = tid % TK;  // reduction column within a stage
    const int rw = tid / TK;  // loader row within one pass

    // A row m0 + rw + RS*q of group g: lane part rw*OHW, the rest uniform.
    // Rows past Kg and taps past R only feed accumulators the epilogue never
    // stores; their loads stay inside the tensors or read 0.
    const uint32_t a_lane4 = (uint32_t)(rw * OHW) * 4u;
    const uint32_t a_soff4 = (uint32_t)((g * p.Kg + m0) * OHW) * 4u;
    const uint32_t b_lane4 = (uint32_t)((lane >> 4) * IHW) * 4u;
    uint32_t b_soff[EB];
    uint32_t b_bit[EB];
#pragma unroll
    for (int q = 0; q < EB; ++q) {
        const int tg = r0 / 4 + wave + 4 * q;
        const int cb = tg / KHW;
        const int t = tg - cb * KHW;
        const int u = t / KW;
        const int v = t - u * KW;
        b_soff[q] = (uint32_t)((g * p.Cg + 4 * cb) * IHW + u * IW + v) * 4u;
        b_bit[q] = (uint32_t)t;
    }

    float rA[EA], rB[EB];
    typedef uint32_t u32x3 __attribute__((ext_vector_type(3)));
    auto load_entry = [&](int cbase) {
        return __builtin_bit_cast(
            u32x3, __builtin_amdgcn_raw_buffer_load_b96(rtab, (uint32_t)(cbase + kc) * 12u, 0, 0));
    };
    auto load_stage = [&](const u32x3& e) {
        const uint32_t db4 = e[2] + a_lane4;
#pragma unroll
        for (int q = 0; q < EA; ++q)
            rA[q] = __builtin_bit_cast(
                float, __builtin_amdgcn_raw_buffer_load_b32(
                           rd, db4, (int)(a_soff4 + (uint32_t)(RS * q * OHW) * 4u), 0));
        const uint32_t xb4 = e[0] + b_lane4;
        const uint32_t nok = e[1];
#pragma unroll
        for (int q = 0; q < EB; ++q)
            rB[q] = __builtin_bit_cast(
                float, __builtin_amdgcn_raw_buffer_load_b32(rx, xb4 | ((nok >> b_bit[q]) << 31),
                                                            (int)b_soff[q], 0));
    };

    // Loader row rw + RS*q is row 32*(q/2) + rw + 16*(q%2) of the tile;
    // rows q and q + 2 of a block pair sit side by side.
    auto store_rows = [&](float* row, const float* vals, auto nsub_tag, auto e_tag) {
        constexpr int NSUB = decltype(nsub_tag)::value;
        constexpr int E = decltype(e_tag)::value;
#pragma unroll
        for (int q = 0; q < E; ++q) {
            const int sub = q / 2;
            const int mi = sub % NSUB;
            const int pos = quad_lds_pos<NSUB>(sub, rw + 16 * (q % 2));
            if ((mi | 1) < NSUB) {
                if ((mi & 1) == 0)
                    *(float2*)&row[pos] = make_float2(vals[q], vals[q + 2]);
            } else {
                row[pos] = vals[q];
            }
        }
    };
    auto store_stage = [&](int buf) {
        store_rows(&As[buf][kc][0], rA, std::integral_constant<int, MI>{},
                   std::integral_constant<int, EA>{});
        store_rows(&Bs[buf][kc][0], rB, std::integral_constant<int, NI>{},
                   std::integral_constant<int, EB>{});
    };

    floatx16 acc[MI][NI];
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int ni = 0; ni < NI; ++ni)
            acc[mi][ni] = floatx16{};

    // bias-gradient partials, as in conv_wgrad_f32_kernel
    const bool want_db = p.dbp != nullptr && rt == 0;
    const int db_pos = quad_lds_pos<MI>(tid / 32, tid % 32);
    float dsum = 0.f;

    const int nst = col_end > col_begin ? (col_end - col_begin + TK - 1) / TK : 0;
    u32x3 e_next = {0u, 0u, 0u};  // table entries of the next stage
    if (nst > 0) {
        load_stage(load_entry(col_begin));
        if (nst > 1)
            e_next = load_entry(col_begin + TK);
        store_stage(0);
    }
    __syncthreads();

    const int kl = lane >> 5;
    const int l32 = lane & 31;
    // Column blocks of this wave that hold taps below R (wave-uniform): the
    // last tap tile of a layer whose R is not a multiple of TN runs no MFMAs
    // for blocks wholly past R, which leaves their SIMD time to the other
    // resident workgroups (CaffeNet conv2: 48 of the last tile's 128 taps are
    // real).  The stage loop below is instantiated once per count.
    const int nbv = __builtin_amdgcn_readfirstlane(
        min(max((p.R - (r0 + wn * NI * MT) + MT - 1) / MT, 0), NI));
    auto stage_loop = [&](auto nb_tag) {
    constexpr int NB = decltype(nb_tag)::value;
    for (int s = 0; s < nst; ++s) {
        const int cur = s & 1;
        if (s + 1 < nst) {
            load_stage(e_next);
            // (unconditional: past the split it reads unused entries, or 0
            // past the table, and the stores below wait for the data only)
            e_next = load_entry(col_begin + (s + 2) * TK);
        }
        if (want_db && tid < TM) {
#pragma unroll
            for (int k = 0; k < TK; ++k)
                dsum += As[cur][k][db_pos];
        }
        constexpr int KS = TK / 2;
        constexpr int PF = 2;
        float fa[PF + 1][MI], fb[PF + 1][NI];
        auto read_frags = [&](const float* row, float* f, auto nsub_tag, int slab) {
            constexpr int NSUB = decltype(nsub_tag)::value;
#pragma unroll
            for (int mi = 0; mi < NSUB; mi += 2) {
                const int pos = quad_lds_pos<NSUB>(slab * NSUB + mi, l32);
                if (mi + 1 < NSUB) {
                    const float2 v = *(const float2*)&row[pos];
                    f[mi] = v.x;
                    f[mi + 1] = v.y;
                } else {
                    f[mi] = row[pos];
                }
            }
        };
        auto read_frag = [&](int ks, int slot) {
            read_frags(&As[cur][2 * ks + kl][0], fa[slot], std::integral_constant<int, MI>{}, wm);
            read_frags(&Bs[cur][2 * ks + kl][0], fb[slot], std::integral_constant<int, NI>{}, wn);
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
                for (int ni = 0; ni < NB; ++ni)
                    acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x2f32(
                        fa[ks % (PF + 1)][mi], fb[ks % (PF + 1)][ni], acc[mi][ni], 0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
        }
        if (s + 1 < nst)
            store_stage(cur ^ 1);
        __syncthreads();
    }
    };
    if (nbv == NI)
        stage_loop(std::integral_constant<int, NI>{});
    else if (NI > 1 && nbv == 1)
        stage_loop(std::integral_constant<int, 1>{});
    else
        stage_loop(std::integral_constant<int, 0>{});

    if (want_db) {
        const int m = m0 + tid;
        if (tid < TM && m < p.Kg)
            p.dbp[split * p.K + g * p.Kg + m] = dsum;
    }

    // Partial P[split][g*Kg + m][r], r = c*KHW + t for r' = (cb*KHW + t)*4 + c % 4.
    const __amdgpu_buffer_rsrc_t rp = make_rsrc(p.P, p.P_bytes);
    const int pbase = split * p.K * p.R;
#pragma unroll
    for (int ni = 0; ni < NI; ++ni) {
        const int rq = r0 + wn * NI * MT + ni * MT + l32;
        const int tg = rq >> 2;
        const int cb = tg / KHW;
        const int r = (4 * cb + (rq & 3)) * KHW + (tg - cb * KHW);
        const bool rok = rq < p.R;
#pragma unroll
        for (int mi = 0; mi < MI; ++mi) {
#pragma unroll
            for (int q = 0; q < 16; ++q) {
                const int m = m0 + wm * MI * MT + mi * MT + 8 * (q >> 2) + 4 * kl + (q & 3);
                const bool ok = rok && m < p.Kg;
                const uint32_t off = ok ? (uint32_t)(pbase + (g * p.Kg + m) * p.R + r) * 4u : kOob;
                buf_st_f32(acc[mi][ni][q], rp, off);
            }
        }
    }
}

// ----------------------------------------------------------- LDS-DMA order
// The quad-order GEMM with both operands copied global -> LDS by the buffer
// unit (one wave instruction writes 64 consecutive floats), with lanes along
// the reduction index: no register staging, no LDS stores, no waits on the
// loads before the stores.
//
// LDS holds each operand as [tile row][16 columns of the stage], one 64-byte
// row per tile row, its four 16-byte chunks permuted: logical chunk c of row
// R sits in slot c ^ wchunk_swz(R).  A fragment read (ds_read_b128: 16 rows,
// one chunk) then touches distinct banks whether the LDS serves 16 lanes of
// 64 banks or 8 lanes of 32 banks per cycle.  The MFMA k index is permuted
// within a stage: lane group kl (lane / 32) takes the stage's columns
// 8 kl + step, so one 16-byte read gives a lane's values for four steps; A
// and B use the same permutation, so each step's sum is unchanged.
//
// A copy moves four tile rows (16 lanes each): lane L holds row 4j + L / 16,
// slot (L / 4) % 4, element L % 4, i.e. the logical column
// 4 ((L / 4 % 4) ^ wchunk_swz(4j + L / 16)) + L % 4.  Copy j = wave + 4q of a
// wave has j % 4 = wave, and wchunk_swz depends on the row only through its
// bits 1..3, so a lane's column is the same in every copy of every stage: it
// loads one column-table entry per stage.
__device__ __forceinline__ int wchunk_swz(int r)
{
    return ((r >> 2) & 1) | ((((r >> 1) ^ (r >> 3)) & 1) << 1);
}

template <int WM, int WN, int MI, int NI, int KH, int KW>
__global__ void __launch_bounds__(64 * WM * WN)
conv_wgrad_dma_f32_kernel(const WgradParams p)
{
    constexpr int MT = 32;
    constexpr int NW = WM * WN;
    constexpr int TM = WM * MI * MT;
    constexpr int TN = WN * NI * MT;
    constexpr int TK = 16;
    constexpr int CA = TM / 4;             // A copies per stage
    constexpr int CB = TN / 4;             // B copies per stage
    constexpr int NA = CA / NW, NB = CB / NW;
    constexpr int KHW = KH * KW;
    static_assert(NW == 4 && CA % NW == 0 && CB % NW == 0, "copy mapping: wave = copy % 4");
    static_assert(KHW < 32, "one mask bit per tap");

    __shared__ float As0[TM * TK], As1[TM * TK];
    __shared__ float Bs0[TN * TK], Bs1[TN * TK];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave % WM;
    const int wn = wave / WM;
    const int n_rt = (p.R + TN - 1) / TN;
    const int n_mt = (p.Kg + TM - 1) / TM;
    const int T = wgrad_tile_index(p, n_rt * n_mt);
    if (T >= n_rt * n_mt * p.G * p.splits)
        return;
    const int rt = T % n_rt;
    const int mt = (T / n_rt) % n_mt;
    const int g = (T / (n_rt * n_mt)) % p.G;
    const int split = T / (n_rt * n_mt * p.G);
    const int m0 = mt * TM;
    const int r0 = rt * TN;
    const int IW = p.IW, IHW = p.IH * p.IW;
    const int OHW = p.OH * p.OW;
    const int col_begin = split * p.cols_per_split;
    const int col_end = min(p.Ncol, col_begin + p.cols_per_split);

    const __amdgpu_buffer_rsrc_t rd = make_rsrc(p.D, p.D_bytes);
    // X through a base p.xpad elements early, as in the quad kernel
    const __amdgpu_buffer_rsrc_t rx =
        make_rsrc((const char*)p.X - 4 * (size_t)p.xpad, p.X_bytes + 4u * (uint32_t)p.xpad);
    const __amdgpu_buffer_rsrc_t rtab = make_rsrc(p.T, p.T_bytes);

    // this lane's place in every copy: row 4j + rg, logical column kcol
    const int rg = lane >> 4;
    const int kcol = 4 * (((lane >> 2) & 3) ^ wchunk_swz(4 * wave + rg)) + (lane & 3);
    // A copy q: rows m0 + 4j .. + 3 of group g, j = wave + 4q (scalar part),
    // the lane's row rg in its lane offset
    const uint32_t a_lane4 = (uint32_t)(rg * OHW) * 4u;
    // B copy q: quad rows r0 + 4j .. + 3 = channels 4 cb .. 4 cb + 3 (the
    // lane's c % 4 = rg) of tap t: offset and mask bit uniform
    const uint32_t b_lane4 = (uint32_t)(rg * IHW) * 4u;
    uint32_t b_soff[NB], b_bit[NB];
#pragma unroll
    for (int q = 0; q < NB; ++q) {
        const int tg = r0 / 4 + wave + NW * q;
        const int cb = tg / KHW;
        const int t = tg - cb * KHW;
        const int u = t / KW;
        const int v = t - u * KW;
        b_soff[q] = (uint32_t)((g * p.Cg + 4 * cb) * IHW + u * IW + v) * 4u;
        b_bit[q] = (uint32_t)t;
    }
    const uint32_t a_soff0 = (uint32_t)((g * p.Kg + m0 + 4 * wave) * OHW) * 4u;
    const uint32_t a_step4 = (uint32_t)(4 * NW * OHW) * 4u;

    typedef uint32_t u32x3 __attribute__((ext_vector_type(3)));
    auto load_entry = [&](int cbase) {
        return __builtin_bit_cast(
            u32x3,
            __builtin_amdgcn_raw_buffer_load_b96(rtab, (uint32_t)(cbase + kcol) * 12u, 0, 0));
    };
    auto copy_stage = [&](float* As, float* Bs, const u32x3& e) {
        const uint32_t da = e[2] + a_lane4;
#pragma unroll
        for (int q = 0; q < NA; ++q)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rd, (lds_void*)&As[16 * 4 * (wave + NW * q)],
                                                     4, da, a_soff0 + q * a_step4, 0, 0);
        const uint32_t xb = e[0] + b_lane4;
#pragma unroll
        for (int q = 0; q < NB; ++q)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (lds_void*)&Bs[16 * 4 * (wave + NW * q)],
                                                     4, xb | ((e[1] >> b_bit[q]) << 31),
                                                     b_soff[q], 0, 0);
    };

    floatx16 acc[MI][NI];
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int ni = 0; ni < NI; ++ni)
            acc[mi][ni] = floatx16{};

    // bias-gradient partials: the first tap tile's threads t < TM add up row t
    const bool want_db = p.dbp != nullptr && rt == 0;
    float dsum = 0.f;

    // fragment reads: tile row R of a 32-row block, chunks 2 kl and 2 kl + 1
    const int l32 = lane & 31;
    const int kl = lane >> 5;
    int fa[MI][2], fb[NI][2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
#pragma unroll
        for (int mi = 0; mi < MI; ++mi) {
            const int R = wm * MI * MT + mi * MT + l32;
            fa[mi][h] = R * TK + 4 * ((2 * kl + h) ^ wchunk_swz(R));
        }
#pragma unroll
        for (int ni = 0; ni < NI; ++ni) {
            const int R = wn * NI * MT + ni * MT + l32;
            fb[ni][h] = R * TK + 4 * ((2 * kl + h) ^ wchunk_swz(R));
        }
    }
    // column blocks of this wave that hold taps below R (as in the quad kernel)
    const int nbv = __builtin_amdgcn_readfirstlane(
        min(max((p.R - (r0 + wn * NI * MT) + MT - 1) / MT, 0), NI));

    const int nst = col_end > col_begin ? (col_end - col_begin + TK - 1) / TK : 0;
    u32x3 e_next = {0u, 0u, 0u};
    if (nst > 0) {
        copy_stage(As0, Bs0, load_entry(col_begin));
        e_next = load_entry(col_begin + TK);
    }
    __builtin_amdgcn_s_waitcnt(kVmcnt0);
    __syncthreads();

    auto stage_loop = [&](auto nb_tag) {
    constexpr int NB_ = decltype(nb_tag)::value;
    for (int s0 = 0; s0 < nst; s0 += 2) {
#pragma unroll
        for (int hb = 0; hb < 2; ++hb) {
            const int s = s0 + hb;
            if (s >= nst)
                break;
            float* Ac = hb ? As1 : As0;
            float* Bc = hb ? Bs1 : Bs0;
            float* An = hb ? As0 : As1;
            float* Bn = hb ? Bs0 : Bs1;
            if (s + 1 < nst) {
                copy_stage(An, Bn, e_next);
                // (past the split it reads unused entries, or 0 past the table)
                e_next = load_entry(col_begin + (s + 2) * TK);
            }
            if (want_db && tid < TM) {
                // row tid in the order of its logical chunks
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const floatx4 v =
                        *(const floatx4*)&Ac[tid * TK + 4 * (c ^ wchunk_swz(tid))];
                    dsum += v[0];
                    dsum += v[1];
                    dsum += v[2];
                    dsum += v[3];
                }
            }
            __builtin_amdgcn_sched_barrier(0);
            floatx4 xa[2][MI], xb[2][NI];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
#pragma unroll
                for (int mi = 0; mi < MI; ++mi)
                    xa[h][mi] = *(const floatx4*)&Ac[fa[mi][h]];
#pragma unroll
                for (int ni = 0; ni < NI; ++ni)
                    xb[h][ni] = *(const floatx4*)&Bc[fb[ni][h]];
            }
#pragma unroll
            for (int h = 0; h < 2; ++h)
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
                        for (int ni = 0; ni < NB_; ++ni)
                            acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x2f32(
                                xa[h][mi][i], xb[h][ni][i], acc[mi][ni], 0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
            // the next stage's copies have landed, for every wave
            __builtin_amdgcn_s_waitcnt(kVmcnt0);
            __syncthreads();
        }
    }
    };
    if (nbv == NI)
        stage_loop(std::integral_constant<int, NI>{});
    else if (NI > 1 && nbv == 1)
        stage_loop(std::integral_constant<int, 1>{});
    else
        stage_loop(std::integral_constant<int, 0>{});

    if (want_db) {
        const int m = m0 + tid;
        if (tid < TM && m < p.Kg)
            p.dbp[split * p.K + g * p.Kg + m] = dsum;
    }

    // Partial P[split][g*Kg + m][r], r = c*KHW + t for r' = (cb*KHW + t)*4 + c % 4.
    const __amdgpu_buffer_rsrc_t rp = make_rsrc(p.P, p.P_bytes);
    const int pbase = split * p.K * p.R;
#pragma unroll
    for (int ni = 0; ni < NI; ++ni) {
        const int rq = r0 + wn * NI * MT + ni * MT + l32;
        const int tg = rq >> 2;
        const int cb = tg / KHW;
        const int r = (4 * cb + (rq & 3)) * KHW + (tg - cb * KHW);
        const bool rok = rq < p.R;
#pragma unroll
        for (int mi = 0; mi < MI; ++mi) {
#pragma unroll
            for (int q = 0; q < 16; ++q) {
                const int m = m0 + wm * MI * MT + mi * MT + 8 * (q >> 2) + 4 * kl + (q & 3);
                const bool ok = rok && m < p.Kg;
                const uint32_t off = ok ? (uint32_t)(pbase + (g * p.Kg + m) * p.R + r) * 4u : kOob;
                buf_st_f32(acc[mi][ni][q], rp, off);
            }
        }
    }
}

// One thread per column: see launch_wgrad_col_table.
__global__ void __launch_bounds__(256)
wgrad_col_table_kernel(uint32_t* __restrict__ T, int ncol, int ncol_pad, int C, int IH, int IW,
                       int K, int OH, int OW, int kh, int kw, int sh, int sw, int ph, int pw)
{
    const int col = blockIdx.x * 256 + threadIdx.x;
    if (col >= ncol_pad)
        return;
    uint32_t e[3] = {kOob, ~0u, kOob};
    if (col < ncol) {
        const int OHW = OH * OW;
        const int n = col / OHW;
        const int pix = col - n * OHW;
        const int i = pix / OW;
        const int j = pix - i * OW;
        const int ih0 = i * sh - ph;
        const int iw0 = j * sw - pw;
        uint32_t nok = 0;
        for (int u = 0; u < kh; ++u)
            for (int v = 0; v < kw; ++v)
                if ((unsigned)(ih0 + u) >= (unsigned)IH || (unsigned)(iw0 + v) >= (unsigned)IW)
                    nok |= 1u << (u * kw + v);
        const int64_t xb = (int64_t)n * C * IH * IW + (int64_t)(ih0 + ph) * IW + (iw0 + pw);
        e[0] = (uint32_t)(xb * 4);
        e[1] = nok;
        e[2] = (uint32_t)(((int64_t)n * K * OHW + pix) * 4);
    }
    T[3 * col] = e[0];
    T[3 * col + 1] = e[1];
    T[3 * col + 2] = e[2];
}

// ------------------------------------------------------------------ launch
namespace {
constexpr int kTK = 16;

struct WTile {
    int wm, wn, mi, ni;
};
constexpr WTile kWTiles[WTILE_COUNT] = {
    {2, 2, 2, 2},  // 128 x 128
    {1, 4, 3, 1},  // 96 x 128
    {2, 2, 1, 2},  // 64 x 128
};

template <int WM, int WN, int MI, int NI, int KH, int KW, int SH, int SW>
hipError_t launch_w(const WgradParams& p, hipStream_t s)
{
    constexpr int TM = WM * MI * 32, TN = WN * NI * 32;
    const int64_t grid = wgrad_grid(p, (int64_t)((p.R + TN - 1) / TN) * ((p.Kg + TM - 1) / TM));
    if (grid > INT_MAX)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL((conv_wgrad_f32_kernel<WM, WN, MI, NI, kTK, KH, KW, SH, SW>),
                       dim3((unsigned)grid), dim3(64 * WM * WN), 0, s, p);
    return hipGetLastError();
}

template <int WM, int WN, int MI, int NI>
hipError_t launch_wg(const WgradParams& p, hipStream_t s)
{
    // compile-time kernels pack their tap table (offsets below 2^22)
    if ((int64_t)p.Cg * p.IH * p.IW >= (int64_t(1) << 22))
        return launch_w<WM, WN, MI, NI, 0, 0, 0, 0>(p, s);
    if (p.sh == 1 && p.sw == 1) {
        if (p.kh == 3 && p.kw == 3)
            return launch_w<WM, WN, MI, NI, 3, 3, 1, 1>(p, s);
        if (p.kh == 5 && p.kw == 5)
            return launch_w<WM, WN, MI, NI, 5, 5, 1, 1>(p, s);
    }
    if (p.kh == 11 && p.kw == 11 && p.sh == 4 && p.sw == 4)
        return launch_w<WM, WN, MI, NI, 11, 11, 4, 4>(p, s);
    return launch_w<WM, WN, MI, NI, 0, 0, 0, 0>(p, s);
}
}  // namespace

int wgrad_tile_m(int tile) { return kWTiles[tile].wm * kWTiles[tile].mi * 32; }
int wgrad_tile_n(int tile) { return kWTiles[tile].wn * kWTiles[tile].ni * 32; }
int wgrad_tile_k() { return kTK; }

hipError_t launch_conv_wgrad_f32(const WgradParams& p, int tile, hipStream_t s)
{
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

namespace {
template <int WM, int WN, int MI, int NI, int KH, int KW>
hipError_t launch_wq(const WgradParams& p, hipStream_t s)
{
    constexpr int TM = WM * MI * 32, TN = WN * NI * 32;
    const int64_t grid = wgrad_grid(p, (int64_t)((p.R + TN - 1) / TN) * ((p.Kg + TM - 1) / TM));
    if (grid > INT_MAX)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL((conv_wgrad_quad_f32_kernel<WM, WN, MI, NI, KH, KW>),
                       dim3((unsigned)grid), dim3(64 * WM * WN), 0, s, p);
    return hipGetLastError();
}

template <int WM, int WN, int MI, int NI>
hipError_t launch_wqg(const WgradParams& p, hipStream_t s)
{
    if (p.kh == 3 && p.kw == 3)
        return launch_wq<WM, WN, MI, NI, 3, 3>(p, s);
    if (p.kh == 5 && p.kw == 5)
        return launch_wq<WM, WN, MI, NI, 5, 5>(p, s);
    return hipErrorInvalidValue;
}
}  // namespace

namespace {
template <int WM, int WN, int MI, int NI, int KH, int KW>
hipError_t launch_wd(const WgradParams& p, hipStream_t s)
{
    constexpr int TM = WM * MI * 32, TN = WN * NI * 32;
    const int64_t grid = wgrad_grid(p, (int64_t)((p.R + TN - 1) / TN) * ((p.Kg + TM - 1) / TM));
    if (grid > INT_MAX)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL((conv_wgrad_dma_f32_kernel<WM, WN, MI, NI, KH, KW>),
                       dim3((unsigned)grid), dim3(64 * WM * WN), 0, s, p);
    return hipGetLastError();
}

template <int WM, int WN, int MI, int NI>
hipError_t launch_wdg(const WgradParams& p, hipStream_t s)
{
    if (p.kh == 3 && p.kw == 3)
        return launch_wd<WM, WN, MI, NI, 3, 3>(p, s);
    if (p.kh == 5 && p.kw == 5)
        return launch_wd<WM, WN, MI, NI, 5, 5>(p, s);
    return hipErrorInvalidValue;
}
}  // namespace

hipError_t launch_conv_wgrad_dma_f32(const WgradParams& p, int tile, hipStream_t s)
{
    if (!wgrad_quad_supported(p.Cg, p.kh, p.kw) || p.T == nullptr || p.xpad < 0 ||
        p.cols_per_split % 16 != 0)
        return hipErrorInvalidValue;
    switch (tile) {
    case WTILE_128x128:
        return launch_wdg<2, 2, 2, 2>(p, s);
    case WTILE_96x128:
        return launch_wdg<1, 4, 3, 1>(p, s);
    case WTILE_64x128:
        return launch_wdg<2, 2, 1, 2>(p, s);
    default:
        return hipErrorInvalidValue;
    }
}

bool wgrad_quad_supported(int Cg, int kh, int kw)
{
    return Cg % 4 == 0 && ((kh == 3 && kw == 3) || (kh == 5 && kw == 5));
}

hipError_t launch_conv_wgrad_quad_f32(const WgradParams& p, int tile, hipStream_t s)
{
    if (!wgrad_quad_supported(p.Cg, p.kh, p.kw) || p.T == nullptr || p.xpad < 0)
        return hipErrorInvalidValue;
    switch (tile) {
    case WTILE_128x128:
        return launch_wqg<2, 2, 2, 2>(p, s);
    case WTILE_96x128:
        return launch_wqg<1, 4, 3, 1>(p, s);
    case WTILE_64x128:
        return launch_wqg<2, 2, 1, 2>(p, s);
    default:
        return hipErrorInvalidValue;
    }
}

hipError_t launch_wgrad_col_table(uint32_t* T, int ncol, int ncol_pad, int C, int IH, int IW,
                                  int K, int OH, int OW, int kh, int kw, int sh, int sw, int ph,
                                  int pw, hipStream_t s)
{
    if (ncol_pad <= 0)
        return hipSuccess;
    if (ncol_pad % 16 != 0 || ncol_pad < ncol || kh * kw >= 32)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(wgrad_col_table_kernel, dim3((unsigned)((ncol_pad + 255) / 256)), dim3(256),
                       0, s, T, ncol, ncol_pad, C, IH, IW, K, OH, OW, kh, kw, sh, sw, ph,
                       pw);
    return hipGetLastError();
}

FastDiv make_fastdiv(uint32_t d)
{
    uint32_t l = 0;
    while ((1ull << l) < d)
        ++l;
    const uint32_t shift = 31 + l;
    const uint64_t mul = ((1ull << shift) + d - 1) / d;
    return FastDiv{d, (uint32_t)mul, shift};
}

}  // namespace caffe_hip
