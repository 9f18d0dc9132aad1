// api.cpp -- the C ABI (include/caffe_conv.h, include/caffe_layers.h):
// argument validation, the workspace plan, and the choice of kernels.  No
// function here touches the GPU before every argument has been checked.
#include <hip/hip_runtime.h>

#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <mutex>

#include "../../include/caffe_conv.h"
#include "../../include/caffe_layers.h"
#include "../../include/caffe_solver.h"
#include "kernels.h"

using namespace caffe_hip;

namespace {

thread_local char g_err[512];

int fail(int status, const char* fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return status;
}

int hip_fail(hipError_t e, const char* what)
{
    return fail(CAFFE_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

constexpr int64_t kMaxTensorBytes = (int64_t(1) << 31) - 1;
constexpr int32_t kMaxSpatial = 16383;  // spatial sizes, kernels and pads
constexpr size_t kWsAlign = 256;

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

// Everything the kernels need to know about one convolution.
struct ConvPlan {
    int N, C, H, W, K, kh, kw, sh, sw, ph, pw, G, relu, dtype;
    int Ho, Wo, Cg, Kg, R;
    int64_t esize;  // bytes per bottom/weight element
    int64_t bottom_elems, top_elems, weight_elems;
    // data gradient (phase-stacked)
    int Th, Tw, a0h, a0w, Ah, Aw, Mt, Rt;
    // weight gradient split-K; the quad-order kernel reads a per-column table
    // of ncol_pad entries at off_coltab
    int splits, cols_per_split, wgrad_tile;
    bool wgrad_quad, wgrad_dma;
    int ncol_pad, xpad;
    size_t off_coltab;
    // reduction order of the implicit GEMMs: tap-major r = (u, v, c) when the
    // gathered channels per group fill whole pipeline stages
    int fwd_tile, dgrad_tile;
    bool fwd_tap, dgrad_tap;
    // channel-major forward: tap-offset table of fwd_rpad entries
    bool fwd_taps;
    int fwd_rpad;
    size_t off_taps_fwd;
    int blocked, xcd_order, wgrad_xcd_order;  // reduction and tile orders (see kernels.h)
    bool wgrad_unit_order;                    // bf16 weight gradient: units per XCD
    int dgrad_blocked;                        // bf16 data gradient: channel-blocked order
    // workspace layout (byte offsets), per pass
    size_t off_d, off_sums, off_wt, off_part;
    size_t ws_fwd, ws_data, ws_weights, ws_both;
    // bf16 operands: channel-contiguous staging with each group's channels
    // padded to a multiple of 8 (Cgp, Kgp), or a single group of at most 4
    // channels padded to Cgp in {1, 2, 4} with 8 / Cgp taps per 16-byte chunk
    // (tpc; kw rounded up to kwp); padded reduction lengths of the forward
    // (Rp) and data-gradient (Rtp) GEMMs; weight-gradient columns Rw
    int Cgp, Kgp, Rp, Rtp, Rw, tpc, kwp;
    // space-to-depth staging of a strided layer (s2d = its stride S, else 0):
    // S x S pixel blocks of the input become channels (Cgp from C * S * S),
    // and the layer a stride-1 one with gkh x kwp kernel taps of the blocks
    // (gkh = ceil(kh / S), kwp = ceil(kw / S)); without it gkh = kh
    int s2d, gkh;
    // zero-bordered bf16 staging: the input on an XHp x XWp grid (real pixels
    // at (ph, pw)), the top gradient on a DHp x DWp grid (real pixels at
    // (dtb, dlb)); the data-gradient gather reads the latter from (doh0, dow0)
    int XHp, XWp, DHp, DWp, dtb, dlb, doh0, dow0;
    int fwd_pipe, dgrad_pipe;       // bf16 GEMM pipelines (Bf16Pipe)
    size_t off_xh_fwd, off_wp_fwd;  // forward: [Xh][Wp]
    size_t off_dh, off_xh;          // backward: [Xh][Dh][sums][Wt][partials] (Xh where the
                                    // forward left it)
    // inner-product shape (1x1 kernel on 1x1 spatial, one group, fp32): dense
    // split-K GEMMs with rows = samples (forward, data gradient) or outputs
    // (weight gradient)
    // split-K of the convolution GEMMs (1 = the fused epilogue): partials
    // after the packed weights (forward) and in the weight-partial region
    // (data gradient)
    int fwd_splits, fwd_sps, dgrad_splits, dgrad_sps;
    size_t off_fwd_part;
    // bf16 data gradient written as the staged top gradient of the layer
    // below (caffe_conv_backward_into), else null
    struct StageTarget {
        uint16_t* Sh;
        float* Ssum;
        uint32_t Sh_bytes, Ssum_bytes;
        int Hp, Wp, tb, lb, Ktot, T;
    };
    const StageTarget* below;
    // tail splits of the forward and data-gradient GEMMs (splits 1: none):
    // the tiles from T on cut into `splits` reduction ranges of sps stages,
    // their partials at the split partials' offset
    struct Tail {
        int T, splits, sps, c0;
        int64_t bytes;
    } fwd_tail, dgrad_tail;
    bool dense;
    int fc_tile_f, fc_tile_d, fc_tile_w;
    int fc_splits_f, fc_sps_f, fc_splits_d, fc_sps_d, fc_splits_w, fc_sps_w;
    size_t fc_off_xt, fc_off_wp, fc_off_pf;  // forward: [X^T][W^T] (C % 4 != 0)[partials]
    size_t fc_off_d, fc_off_dt, fc_off_pb;   // backward: [D][D^T][partials]
};

// bf16 products (CAFFE_BF16 and CAFFE_BF16_F32_BOTTOM), and a float bottom
// (CAFFE_F32, and CAFFE_BF16_F32_BOTTOM, which rounds it while staging)
bool is_bf16(const ConvPlan& q) { return q.dtype != CAFFE_F32; }
bool bottom_f32(const ConvPlan& q) { return q.dtype != CAFFE_BF16; }

// Split-K plan of a dense GEMM with M rows, ncol columns and a reduction of R
// on `cus` compute units.  Workgroups are dealt evenly to the units and a
// unit works through its share at its MFMA rate, so the GEMM takes about
// ceil(tiles * s / cus) * ceil(stages / s) workgroup-stages of time (measured
// on the inner-product shapes: splits that leave some units one workgroup
// more than the rest cost that whole extra workgroup; a unit with a single
// workgroup runs it ~10% slower, its memory latency less hidden); s splits
// add s * groups * M * ncol partial sums written and read back once.  The
// plan takes the s with the least modelled time (ties: fewer splits), and
// splits only when that time is at least 10% below the unsplit one.
void plan_splits(int M, int ncol, int R, int tile, int cus, int forced, int* splits, int* sps,
                 int groups = 1)
{
    const int tm = gemm_tile_m(tile), tn = gemm_tile_n(tile), tk = gemm_tile_k(tile);
    const int64_t tiles = std::max<int64_t>(
        1, (int64_t)groups * ((M + tm - 1) / tm) * ((ncol + tn - 1) / tn));
    const int64_t nst = std::max(1, (R + tk - 1) / tk);
    cus = std::max(1, cus);
    // one workgroup-stage at ~85% of a unit's fp32 MFMA rate (157.3 TFLOP/s
    // over 256 units), partials at ~4 TB/s
    const double t_stage = 2.0 * tm * tn * tk / (0.85 * 157.3e12 / 256);
    const double t_byte = 1.0 / 4e12;
    int64_t best = 1;
    double best_t = -1, t1 = 0;
    for (int64_t sp = 1; sp <= nst; ++sp) {
        const double part = sp > 1 ? 8.0 * sp * groups * M * ncol : 0.0;
        if (part / 2 > (double)kMaxTensorBytes)
            break;
        const int64_t load = (tiles * sp + cus - 1) / cus;  // workgroups per unit
        const double t = (double)load * ((nst + sp - 1) / sp) * t_stage * (load == 1 ? 1.1 : 1.0) +
                         part * t_byte;
        if (sp == 1)
            t1 = t;
        if (best_t < 0 || t < best_t * (1 - 1e-9)) {
            best = sp;
            best_t = t;
        }
    }
    // split only for a clear modelled gain (the model ignores the reduce's
    // launch and its read of the partials' first split)
    if (best > 1 && best_t > 0.9 * t1)
        best = 1;
    if (forced > 0)  // profiling only
        best = std::min<int64_t>(forced, nst);
    *sps = (int)((nst + best - 1) / best);
    *splits = (int)((nst + *sps - 1) / *sps);
}

// Tail split of a GEMM with G groups of M x ncol outputs on a tile and a
// reduction of R (one workgroup per tile otherwise).  When the tiles do not
// deal evenly to the `cus` compute units, some units run one workgroup more
// than the rest while the others idle (CaffeNet N=256: conv5's forward and
// conv3's data gradient have 676 128 x 128 tiles, 2.64 per unit, and run
// ~20% longer than conv3's forward with 1014, 3.96 per unit).  The last
// tiles past whole rounds of the units -- whole column tiles of the last
// group -- are then cut into s reduction ranges, one workgroup each, whose
// partials a reduce adds: every unit gets about the same work.  The model:
// workgroup b runs on unit b % cus, a unit's time is the sum of its
// workgroups' stages; s (2..8) is taken when the modelled time with the
// partial sums' traffic (written and read once at ~4 TB/s, plus ~6 us for
// the reduce) beats the plain grid's by 1.5% or more (measured alone at
// N=256: conv5's forward 0.362 -> 0.348 ms with 3 ranges, conv3's data
// gradient 0.719 -> 0.661, conv2's forward 0.929 -> 0.908 with 2, conv2's
// data gradient 1.032 -> 0.993 with 4; conv1's data gradient, which the
// model leaves whole, 0.630 -> 0.652 with 2).
void plan_tail(int M, int64_t ncol, int R, int tile, int G, int cus, int forced, int forced_cus,
               ConvPlan::Tail* t)
{
    *t = ConvPlan::Tail{0, 1, 0, 0, 0};
    const int tm = gemm_tile_m(tile), tn = gemm_tile_n(tile), tk = gemm_tile_k(tile);
    const int64_t n_mt = (M + tm - 1) / tm, n_ct = (ncol + tn - 1) / tn;
    const int64_t n_tiles = n_mt * n_ct * G;
    const int64_t nst = (R + tk - 1) / tk;
    if (forced_cus > 0)  // profiling and tests only
        cus = forced_cus;
    cus = std::max(1, cus);
    if (forced == 0 || n_tiles < cus || nst < 8 || M <= 0)
        return;
    const int64_t past = n_tiles % cus;
    if (past == 0 && forced < 0)
        return;
    // whole column tiles of the last group
    const int64_t n_tail = std::max<int64_t>(n_mt, (past + n_mt - 1) / n_mt * n_mt);
    if (n_tail > n_mt * n_ct)
        return;
    const int64_t full = n_tiles - n_tail;
    const double t_stage = 2.0 * tm * tn * tk / (0.8 * 157.3e12 / 256);
    auto unit_time = [&](int64_t s) {  // the busiest unit's stages
        const int64_t sps = (nst + s - 1) / s;
        int64_t worst = 0;
        for (int64_t c = 0; c < cus; ++c) {
            const int64_t nf = full > c ? (full - 1 - c) / cus + 1 : 0;
            // partial workgroups b = full .. full + n_tail * s - 1 on unit c
            const int64_t lo = full, hi = full + n_tail * s;
            const int64_t first = lo + ((c - lo % cus) % cus + cus) % cus;
            const int64_t np = first < hi ? (hi - 1 - first) / cus + 1 : 0;
            worst = std::max(worst, nf * nst + np * sps);
        }
        return worst;
    };
    const double plain = (double)((n_tiles + cus - 1) / cus) * nst * t_stage;
    double best_t = plain * 0.985;
    int64_t best = 0;
    for (int64_t s = 2; s <= 8; ++s) {
        const int64_t sps = (nst + s - 1) / s;
        if (sps < 4 || (s - 1) * sps >= nst)
            continue;
        const int64_t bytes = s * (int64_t)M * (ncol - (n_ct - n_tail / n_mt) * tn) * 4;
        const double tt = unit_time(s) * t_stage + 2.0 * bytes / 4e12 + 6e-6;
        if (forced > 1 ? s == forced : tt < best_t) {
            best_t = tt;
            best = s;
        }
    }
    if (best < 2)
        return;
    t->T = (int)full;
    t->splits = (int)best;
    t->sps = (int)((nst + best - 1) / best);
    t->c0 = (int)((n_ct - n_tail / n_mt) * tn);
    t->bytes = best * (int64_t)M * (ncol - t->c0) * 4;
}

// Tile for a GEMM with M rows: the least padding of M; ties go to the first
// tile of the preference order (measured on CaffeNet's 192-row GEMMs at
// N=256: 64-row tiles beat 96-row ones by 4% in the forward pass and by 13%
// in the data gradient).  `forced` >= 0 picks a tile (profiling only).
int pick_tile(int M, int forced)
{
    if (forced >= 0 && forced < TILE_COUNT)
        return forced;
    static const int order[] = {TILE_128x128, TILE_64x256, TILE_96x256, TILE_48x256};
    int best = order[0];
    double best_waste = 1e30;
    for (int i = 0; i < 4; ++i) {
        const int t = order[i];
        const int tm = gemm_tile_m(t);
        const double waste = (double)((M + tm - 1) / tm * tm) / M;
        if (waste < best_waste - 1e-9) {
            best = t;
            best_waste = waste;
        }
    }
    return best;
}

// Dense (inner-product) GEMM tile for M rows: 128 x 128 unless it pads M by
// more than 5% (measured: on 1000 rows it beats the 48-row tile's lesser
// padding), else the forward pass's choice.
int pick_dense_tile(int M, int forced)
{
    if (forced >= 0 && forced < TILE_COUNT && forced != TILE_128x128_K32)
        return forced;
    if ((double)((M + 127) / 128 * 128) <= 1.05 * M)
        return TILE_128x128;
    return pick_tile(M, -1);
}

// Weight-gradient tile: the least padding of Kg, then the taller tile.
int pick_wgrad_tile(int Kg, int forced)
{
    if (forced >= 0 && forced < WTILE_COUNT)
        return forced;
    int best = WTILE_128x128;
    double best_waste = 1e30;
    for (int t = 0; t < WTILE_COUNT; ++t) {
        const int tm = wgrad_tile_m(t);
        const double waste = (double)((Kg + tm - 1) / tm * tm) / Kg;
        if (waste < best_waste - 1e-9 ||
            (waste < best_waste + 1e-9 && tm > wgrad_tile_m(best))) {
            best = t;
            best_waste = waste;
        }
    }
    return best;
}

// Profiling override of a tuning choice (tile index, split count, kernel
// variant): an integer from the environment, -1 when unset.  The variables
// are read only while CAFFE_PROFILE_OVERRIDES=1 is set, so that a stray
// CAFFE_* variable cannot change what a default call runs (the kernel, the
// split count and with it the summation order).
bool overrides_enabled()
{
    const char* v = getenv("CAFFE_PROFILE_OVERRIDES");
    return v && v[0] == '1' && v[1] == '\0';
}

int env_tile(const char* name)
{
    if (!overrides_enabled())
        return -1;
    const char* v = getenv(name);
    return v && *v ? atoi(v) : -1;
}

int round_up(int x, int a) { return (x + a - 1) / a * a; }

// bf16 weight-gradient tile for Kg output channels per group: the least row
// padding, ties to 128 rows.
int pick_bf16_wgrad_tile(int Kg, int forced)
{
    if (forced >= 0 && forced < BWTILE_COUNT)
        return forced;
    const int64_t r128 = (int64_t)(Kg + 127) / 128 * 128, r96 = (int64_t)(Kg + 95) / 96 * 96;
    return r96 < r128 ? BWTILE_96x256 : BWTILE_128x256;
}

// bf16 GEMM pipeline for a tile: three LDS buffers (copies two stages ahead)
// unless double buffering lets two workgroups share a compute unit's LDS
// (measured on the CaffeNet layers: the 48-row data-gradient tiles gain more
// from the second workgroup than from the deeper pipeline; the 96- and
// 128-row tiles, one workgroup per unit either way, gain from the depth).
int pick_bf16_pipe(int tile)
{
    const int bytes2 = (bf16_tile_m(tile) + 256) * kBf16TK * 2 * 2;
    return 2 * bytes2 <= 160 * 1024 ? BPIPE_2 : BPIPE_3;
}

// bf16 GEMM tile for M rows: the least row padding, ties to the earlier of
// 128, 64, 96, 48 rows (CaffeNet's 192-row GEMMs at N=512: the 64-row tile
// 12-15% faster than the 96-row one).
int pick_bf16_tile(int M, int forced)
{
    if (forced >= 0 && forced < BTILE_COUNT)
        return forced;
    static const int order[] = {BTILE_128x256, BTILE_64x256, BTILE_96x256, BTILE_48x256};
    int best = order[0];
    int64_t best_rows = INT64_MAX;
    for (int t : order) {
        const int tm = bf16_tile_m(t);
        const int64_t rows = (int64_t)(M + tm - 1) / tm * tm;
        if (rows < best_rows) {
            best = t;
            best_rows = rows;
        }
    }
    return best;
}

// The bf16-operand plan: staging sizes, padded reductions, the weight-gradient
// split and the workspace layout.  Called by plan_conv once the common fields
// are set.
int plan_bf16(ConvPlan* p)
{
    ConvPlan& q = *p;
    // Channels per staged group.  A 16-byte chunk of the reduction is 8
    // channels of one tap, or, for one group of at most 4 channels, 8 / Cgp
    // horizontally adjacent taps of Cgp channels: 8 consecutive staged
    // elements, 16-byte aligned when the horizontal stride and the staged
    // width are multiples of the taps per chunk (CaffeNet's conv1: 3 -> 4
    // channels instead of 8).
    q.Cgp = round_up(q.Cg, 8);
    if (q.G == 1)
        for (int c = 1; c <= 4; c *= 2)
            if (c >= q.Cg && q.sw % (8 / c) == 0) {
                q.Cgp = c;
                break;
            }
    q.tpc = q.Cgp < 8 ? 8 / q.Cgp : 1;
    q.kwp = round_up(q.kw, q.tpc);
    q.gkh = q.kh;
    q.s2d = 0;
    q.Kgp = round_up(q.Kg, 8);
    // The staged copies carry the gathers' zero padding as a border: the
    // input's covers every forward tap, the top gradient's every tap of the
    // phase-stacked data-gradient gather (whose padding Th - 1 - a0h may be
    // negative: then the gather starts doh0 rows into the grid instead).
    q.XHp = std::max(q.ph + q.H, (q.Ho - 1) * q.sh + q.kh);
    q.XWp = round_up(std::max(q.pw + q.W, (q.Wo - 1) * q.sw + q.kwp), q.tpc);
    // A strided layer with few channels (CaffeNet's conv1: 3 channels,
    // stride 4) staged space-to-depth when that pads its reduction less:
    // conv1's 11 x 11 x 3 taps become 3 x 3 taps of 48 channels, 432 staged
    // reduction elements (448 padded) instead of 11 x 12 x 4 = 528 (576).
    {
        const int S = q.sh;
        const int cs = round_up(q.C * S * S, 8);
        const int gkh = (q.kh + S - 1) / S, gkw = (q.kw + S - 1) / S;
        const int xhp = q.Ho + gkh - 1, xwp = q.Wo + gkw - 1;
        const int64_t r_plain = ((int64_t)q.kh * q.kwp * q.Cgp + kBf16TK - 1) / kBf16TK;
        const int64_t r_s2d = ((int64_t)gkh * gkw * cs + kBf16TK - 1) / kBf16TK;
        if (q.G == 1 && S >= 2 && q.sw == S && q.kh >= S && q.kw >= S && q.C * S * S <= 64 &&
            r_s2d < r_plain && xhp <= 65535 && q.N <= 65535 &&
            (int64_t)q.C * S * xwp * S * 2 <= 64 * 1024 &&
            (int64_t)q.C * q.H * q.W * 4 < (int64_t(1) << 31)) {
            q.s2d = S;
            q.Cgp = cs;
            q.tpc = 1;
            q.gkh = gkh;
            q.kwp = gkw;
            q.XHp = xhp;
            q.XWp = xwp;
        }
    }
    const int khw = q.gkh * q.kwp;
    const int php = q.Th - 1 - q.a0h, pwp = q.Tw - 1 - q.a0w;
    q.dtb = std::max(php, 0);
    q.dlb = std::max(pwp, 0);
    q.doh0 = q.dtb - php;
    q.dow0 = q.dlb - pwp;
    q.DHp = std::max(q.dtb + q.Ho, q.Ah + q.Th - 1 + q.doh0);
    q.DWp = std::max(q.dlb + q.Wo, q.Aw + q.Tw - 1 + q.dow0);
    const int64_t xh = (int64_t)q.N * q.XHp * q.XWp * q.G * q.Cgp * 2;
    const int64_t dh = (int64_t)q.N * q.DHp * q.DWp * q.G * q.Kgp * 2;
    const int64_t rp = ((int64_t)khw * q.Cgp + kBf16TK - 1) / kBf16TK * kBf16TK;
    const int64_t rtp = ((int64_t)q.Th * q.Tw * q.Kgp + kBf16TK - 1) / kBf16TK * kBf16TK;
    const int64_t rw = (int64_t)khw * q.Cgp;
    const int64_t wp = (int64_t)q.K * rp * 2;
    const int64_t wt = (int64_t)q.G * q.Mt * rtp * 2;
    if (xh > kMaxTensorBytes || dh > kMaxTensorBytes || wp > kMaxTensorBytes ||
        wt > kMaxTensorBytes || rw * q.K * 4 > kMaxTensorBytes)
        return fail(CAFFE_ERR_UNSUPPORTED, "bf16 staging buffers reach 2^31 bytes");
    q.Rp = (int)rp;
    q.Rtp = (int)rtp;
    q.Rw = (int)rw;

    // weight-gradient split-K over the output pixels, as for fp32
    const int64_t ncol = (int64_t)q.N * q.Ho * q.Wo;
    const int tk = kBf16WgradTK;
    q.wgrad_tile = pick_bf16_wgrad_tile(q.Kg, env_tile("CAFFE_BF16_WGRAD_TILE"));
    const int wtm = bf16_wgrad_tile_m(q.wgrad_tile), wtn = kBf16WgradTN;
    const int64_t tiles = (int64_t)((q.Kg + wtm - 1) / wtm) * ((q.Rw + wtn - 1) / wtn) * q.G;
    // one workgroup per compute unit at a time (its LDS): about two rounds
    const int64_t target = env_tile("CAFFE_CONV_WGRAD_BLOCKS") > 0
                               ? env_tile("CAFFE_CONV_WGRAD_BLOCKS")
                               : 2 * (int64_t)device_cu_count();
    int64_t splits = (target + tiles - 1) / tiles;
    const int64_t max_splits = std::max<int64_t>(1, ncol / (8 * tk));
    const int64_t max_by_bytes = std::max<int64_t>(1, kMaxTensorBytes / (rw * q.K * 4));
    // Unit order (see WgradBf16Params::unit_order) where a (group, split)
    // unit holds at least 7 tiles: measured on the CaffeNet layers at N=512,
    // each unit's slab then comes from HBM once instead of once per tile
    // (conv3-5: 4-6x fewer bytes); with fewer tiles per unit (conv1, conv2)
    // the linear order was as fast or faster.  The split count then becomes
    // a multiple of 8 / gcd(G, 8), so that every XCD takes as many units.
    const int64_t per_unit = tiles / q.G;
    const int uo = env_tile("CAFFE_BF16_WGRAD_UNIT_ORDER");
    q.wgrad_unit_order = uo >= 0 ? uo != 0 : per_unit >= 7;
    if (q.wgrad_unit_order) {
        const int64_t m = q.G % 8 == 0 ? 1 : q.G % 4 == 0 ? 2 : q.G % 2 == 0 ? 4 : 8;
        splits = std::max<int64_t>(m, (splits + m / 2) / m * m);
    }
    splits = std::max<int64_t>(1, std::min(std::min(splits, max_splits), max_by_bytes));
    int64_t cps = (ncol + splits - 1) / splits;
    cps = std::max<int64_t>(tk, (cps + tk - 1) / tk * tk);
    splits = std::max<int64_t>(1, (ncol + cps - 1) / cps);
    q.splits = (int)splits;
    q.cols_per_split = (int)cps;
    const int64_t part_bytes = splits * rw * q.K * 4;
    if (part_bytes > kMaxTensorBytes)
        return fail(CAFFE_ERR_UNSUPPORTED, "weight-gradient partials reach 2^31 bytes");

    // data gradient in the channel-blocked reduction order (64-channel blocks
    // of the top gradient outer, taps inner) where the channels allow it
    {
        const int bo = env_tile("CAFFE_BF16_DGRAD_BLOCKED");
        const bool ok = q.Kgp % 64 == 0 && q.Th * q.Tw > 1;
        q.dgrad_blocked = ok && bo != 0 ? 1 : 0;
    }
    q.fwd_tile = pick_bf16_tile(q.Kg, env_tile("CAFFE_BF16_FWD_TILE"));
    q.dgrad_tile = pick_bf16_tile(q.Mt, env_tile("CAFFE_BF16_DGRAD_TILE"));
    const int pipe = env_tile("CAFFE_BF16_PIPE");
    q.fwd_pipe = pipe >= 0 && pipe < BPIPE_COUNT ? pipe : pick_bf16_pipe(q.fwd_tile);
    q.dgrad_pipe = pipe >= 0 && pipe < BPIPE_COUNT ? pipe : pick_bf16_pipe(q.dgrad_tile);
    q.xcd_order = env_tile("CAFFE_CONV_XCD_ORDER") != 0;

    q.off_xh_fwd = 0;
    q.off_wp_fwd = align_up(xh, kWsAlign);
    q.ws_fwd = q.off_wp_fwd + align_up(wp, kWsAlign);
    // bias-gradient partials of the top-gradient staging (and room for the
    // per-image sums of the bias-only pass)
    // (or the partial sums a layer above stages with its data gradient)
    const int64_t terms =
        std::max<int64_t>(std::max<int64_t>(diff_prep_terms(q.N, q.DHp * q.DWp), q.N),
                          stage_below_terms((int64_t)q.N * q.Ho * q.Wo));
    const size_t sums_bytes = align_up((size_t)terms * q.K * 4, kWsAlign);
    if ((int64_t)sums_bytes > kMaxTensorBytes)
        return fail(CAFFE_ERR_UNSUPPORTED, "bias partials reach 2^31 bytes");
    q.off_xh = 0;
    q.off_dh = align_up(xh, kWsAlign);
    q.off_sums = q.off_dh + align_up(dh, kWsAlign);
    q.off_wt = q.off_sums + sums_bytes;
    q.off_part = q.off_wt + align_up(wt, kWsAlign);
    q.ws_data = q.off_part;
    q.ws_weights = q.off_part + align_up(part_bytes, kWsAlign);
    q.ws_both = q.ws_weights;
    return CAFFE_OK;
}

int plan_conv(const caffe_conv_desc* d, ConvPlan* p)
{
    if (!d)
        return fail(CAFFE_ERR_INVALID_ARG, "desc is NULL");
    if (d->N < 0 || d->C < 1 || d->H < 1 || d->W < 1 || d->K < 1)
        return fail(CAFFE_ERR_INVALID_ARG, "blob dims must be >= 1 (N >= 0): N=%d C=%d H=%d W=%d K=%d",
                    d->N, d->C, d->H, d->W, d->K);
    if (d->kernel_h < 1 || d->kernel_w < 1 || d->stride_h < 1 || d->stride_w < 1 ||
        d->pad_h < 0 || d->pad_w < 0)
        return fail(CAFFE_ERR_INVALID_ARG, "kernel/stride must be >= 1 and pad >= 0");
    if (d->group < 1 || d->C % d->group || d->K % d->group)
        return fail(CAFFE_ERR_INVALID_ARG, "group %d must divide C=%d and K=%d", d->group, d->C,
                    d->K);
    if (d->group > 65535)
        return fail(CAFFE_ERR_UNSUPPORTED, "group must be <= 65535");
    if (d->relu != 0 && d->relu != 1)
        return fail(CAFFE_ERR_INVALID_ARG, "relu must be 0 or 1");
    if (d->dtype != CAFFE_F32 && d->dtype != CAFFE_BF16 && d->dtype != CAFFE_BF16_F32_BOTTOM)
        return fail(CAFFE_ERR_UNSUPPORTED, "unknown dtype %d", d->dtype);
    if (d->H + 2 * (int64_t)d->pad_h < d->kernel_h || d->W + 2 * (int64_t)d->pad_w < d->kernel_w)
        return fail(CAFFE_ERR_INVALID_ARG, "kernel larger than the padded input");
    if (d->H > kMaxSpatial || d->W > kMaxSpatial || d->kernel_h > kMaxSpatial ||
        d->kernel_w > kMaxSpatial || d->pad_h > kMaxSpatial || d->pad_w > kMaxSpatial ||
        d->stride_h > kMaxSpatial || d->stride_w > kMaxSpatial)
        return fail(CAFFE_ERR_UNSUPPORTED, "spatial sizes, kernels, strides and pads must be <= %d",
                    kMaxSpatial);

    ConvPlan& q = *p;
    q = ConvPlan{};
    q.N = d->N; q.C = d->C; q.H = d->H; q.W = d->W; q.K = d->K;
    q.kh = d->kernel_h; q.kw = d->kernel_w; q.sh = d->stride_h; q.sw = d->stride_w;
    q.ph = d->pad_h; q.pw = d->pad_w; q.G = d->group; q.relu = d->relu; q.dtype = d->dtype;
    q.Ho = (q.H + 2 * q.ph - q.kh) / q.sh + 1;
    q.Wo = (q.W + 2 * q.pw - q.kw) / q.sw + 1;
    q.Cg = q.C / q.G;
    q.Kg = q.K / q.G;
    q.esize = is_bf16(q) ? 2 : 4;

    const int64_t R = (int64_t)q.Cg * q.kh * q.kw;
    q.bottom_elems = (int64_t)q.N * q.C * q.H * q.W;
    q.top_elems = (int64_t)q.N * q.K * q.Ho * q.Wo;
    q.weight_elems = (int64_t)q.K * R;
    if (q.bottom_elems * 4 > kMaxTensorBytes || q.top_elems * 4 > kMaxTensorBytes ||
        q.weight_elems * 4 > kMaxTensorBytes)
        return fail(CAFFE_ERR_UNSUPPORTED, "a tensor reaches 2^31 bytes");
    q.R = (int)R;

    // Phase-stacked data gradient: output row h with h + ph = sh*a + fh takes
    // the taps u = fh + sh*t of output row i = a - t, t < Th = ceil(kh / sh).
    q.Th = (q.kh + q.sh - 1) / q.sh;
    q.Tw = (q.kw + q.sw - 1) / q.sw;
    q.a0h = q.ph / q.sh;
    q.a0w = q.pw / q.sw;
    q.Ah = (q.H - 1 + q.ph) / q.sh - q.a0h + 1;
    q.Aw = (q.W - 1 + q.pw) / q.sw - q.a0w + 1;
    q.Mt = q.Cg * q.sh * q.sw;
    q.Rt = q.Kg * q.Th * q.Tw;
    const int64_t wt_elems = (int64_t)q.G * q.Mt * q.Rt;
    const int64_t dcols = (int64_t)q.N * q.Ah * q.Aw;
    if (wt_elems * 4 > kMaxTensorBytes || dcols > (int64_t(1) << 30))
        return fail(CAFFE_ERR_UNSUPPORTED, "data-gradient operands reach 2^31 bytes");

    // Weight-gradient split-K: the tile with the least padding of Kg, then
    // enough splits of the reduction for ~`target` workgroups (8 per CU by
    // default), each split at least 8 stages deep.
    const int64_t ncol = (int64_t)q.N * q.Ho * q.Wo;
    const int tk = wgrad_tile_k();
    q.wgrad_tile = pick_wgrad_tile(q.Kg, env_tile("CAFFE_CONV_WGRAD_TILE"));
    const int wtm = wgrad_tile_m(q.wgrad_tile), wtn = wgrad_tile_n(q.wgrad_tile);
    const int64_t tiles = (int64_t)((q.Kg + wtm - 1) / wtm) * ((q.R + wtn - 1) / wtn) * q.G;
    const int64_t target = env_tile("CAFFE_CONV_WGRAD_BLOCKS") > 0
                               ? env_tile("CAFFE_CONV_WGRAD_BLOCKS")
                               : 2048;
    int64_t splits = (target + tiles - 1) / tiles;
    const int64_t max_splits = std::max<int64_t>(1, ncol / (8 * tk));
    const int64_t max_by_bytes = std::max<int64_t>(1, kMaxTensorBytes / (q.weight_elems * 4));
    // unit order (WgradParams::unit_order): splits a multiple of 8 / gcd(G, 8)
    q.wgrad_unit_order = env_tile("CAFFE_CONV_WGRAD_UNIT_ORDER") > 0;
    if (q.wgrad_unit_order) {
        const int64_t m = q.G % 8 == 0 ? 1 : q.G % 4 == 0 ? 2 : q.G % 2 == 0 ? 4 : 8;
        splits = std::max<int64_t>(m, (splits + m / 2) / m * m);
    }
    splits = std::max<int64_t>(1, std::min(std::min(splits, max_splits), max_by_bytes));
    int64_t cps = (ncol + splits - 1) / splits;
    cps = std::max<int64_t>(tk, (cps + tk - 1) / tk * tk);
    splits = std::max<int64_t>(1, (ncol + cps - 1) / cps);
    q.splits = (int)splits;
    q.cols_per_split = (int)cps;
    const int64_t part_bytes = splits * q.weight_elems * 4;
    if (part_bytes > kMaxTensorBytes)
        return fail(CAFFE_ERR_UNSUPPORTED, "weight-gradient partials reach 2^31 bytes");

    q.fwd_tile = pick_tile(q.Kg, env_tile("CAFFE_CONV_FWD_TILE"));
    q.dgrad_tile = pick_tile(q.Mt, env_tile("CAFFE_CONV_DGRAD_TILE"));
    // defaults from measurement: the channel-blocked order and the XCD tile
    // order help the forward / data-gradient GEMMs; the weight gradient keeps
    // the linear tile order (its split partials gain nothing from it)
    q.blocked = env_tile("CAFFE_CONV_BLOCKED") != 0;
    q.xcd_order = env_tile("CAFFE_CONV_XCD_ORDER") != 0;
    q.wgrad_xcd_order = env_tile("CAFFE_CONV_WGRAD_XCD_ORDER") > 0;
    // quad-order weight gradient: its scalar offsets (tap planes, rows of the
    // tile) ride on lane offsets of up to the tensor's size, so both sums
    // must stay below 2^31 with a tile's rows past the end
    {
        const int64_t ihw = (int64_t)q.H * q.W, ohw = (int64_t)q.Ho * q.Wo;
        q.xpad = q.ph * q.W + q.pw;
        const int64_t xlim = q.bottom_elems * 4 + 4 * (int64_t)q.xpad + (q.C + 512) * ihw * 4;
        const int64_t dlim = q.top_elems * 4 + (q.K + 512) * ohw * 4;
        q.wgrad_quad = env_tile("CAFFE_CONV_WGRAD_QUAD") != 0 &&
                       wgrad_quad_supported(q.Cg, q.kh, q.kw) && xlim < kMaxTensorBytes &&
                       dlim < kMaxTensorBytes;
        q.ncol_pad = (int)((ncol + 15) / 16 * 16);
        // the quad order with both operands copied by LDS DMA (the same
        // table and conditions; splits are whole 16-column stages)
        q.wgrad_dma = q.wgrad_quad && env_tile("CAFFE_CONV_WGRAD_DMA") != 0;
    }
    q.fwd_tap = q.Cg % gemm_tile_k(q.fwd_tile) == 0;
    q.dgrad_tap = q.Kg % gemm_tile_k(q.dgrad_tile) == 0;
    q.ws_fwd = align_up(q.weight_elems * 4, kWsAlign);  // the packed weights

    q.dense = false;
    q.fwd_splits = q.dgrad_splits = 1;
    q.fwd_sps = q.dgrad_sps = 0;
    q.off_fwd_part = 0;
    if (is_bf16(q))
        return plan_bf16(&q);

    q.dense = q.H == 1 && q.W == 1 && q.kh == 1 && q.kw == 1 && q.ph == 0 && q.pw == 0 &&
              q.G == 1;
    if (q.dense) {
        // forward: Y[n][k] = sum_c X^T[c][n] W^T[c][k]; data gradient:
        // dX[n][c] = sum_k D^T[k][n] W[k][c]; weight gradient:
        // dW[k][c] = sum_n D[n][k] X[n][c]
        const int N = q.N, C = q.C, K = q.K;
        q.fc_tile_f = pick_dense_tile(std::max(N, 1), env_tile("CAFFE_FC_TILE_F"));
        q.fc_tile_d = pick_dense_tile(std::max(N, 1), env_tile("CAFFE_FC_TILE_D"));
        q.fc_tile_w = pick_dense_tile(K, env_tile("CAFFE_FC_TILE_W"));
        plan_splits(N, K, C, q.fc_tile_f, device_cu_count(),
                    env_tile("CAFFE_FC_SPLITS_F"), &q.fc_splits_f, &q.fc_sps_f);
        plan_splits(N, C, K, q.fc_tile_d, device_cu_count(),
                    env_tile("CAFFE_FC_SPLITS_D"), &q.fc_splits_d, &q.fc_sps_d);
        plan_splits(K, C, N, q.fc_tile_w, device_cu_count(),
                    env_tile("CAFFE_FC_SPLITS_W"), &q.fc_splits_w, &q.fc_sps_w);
        const int64_t pf = (int64_t)q.fc_splits_f * N * K * 4;
        const int64_t pb = std::max((int64_t)q.fc_splits_d * N * C, (int64_t)q.fc_splits_w * K * C) * 4;
        if (pf > kMaxTensorBytes || pb > kMaxTensorBytes)
            return fail(CAFFE_ERR_UNSUPPORTED, "inner-product partials reach 2^31 bytes");
        // the forward stages X^T and W^T only when C % 4 != 0 (the
        // reduction-contiguous GEMM reads 16-byte chunks of rows of C floats)
        const bool staged = C % 4 != 0;
        q.fc_off_xt = 0;
        q.fc_off_wp = staged ? align_up((size_t)N * C * 4, kWsAlign) : 0;
        q.fc_off_pf = staged ? q.fc_off_wp + align_up((size_t)K * C * 4, kWsAlign) : 0;
        q.ws_fwd = q.fc_off_pf + align_up(pf, kWsAlign);
        q.fc_off_d = 0;
        q.fc_off_dt = align_up((size_t)N * K * 4, kWsAlign);
        q.fc_off_pb = q.fc_off_dt + align_up((size_t)N * K * 4, kWsAlign);
        q.ws_data = q.ws_weights = q.ws_both = q.fc_off_pb + align_up(pb, kWsAlign);
        return CAFFE_OK;
    }

    // Split-K of the forward and data-gradient GEMMs for grids too small to
    // fill the device (small batches, long reductions).
    const int cus = device_cu_count();
    plan_splits(q.Kg, q.N * q.Ho * q.Wo, q.R, q.fwd_tile, cus, env_tile("CAFFE_CONV_FWD_SPLITS"),
                &q.fwd_splits, &q.fwd_sps, q.G);
    plan_splits(q.Mt, (int)dcols, q.Rt, q.dgrad_tile, cus, env_tile("CAFFE_CONV_DGRAD_SPLITS"),
                &q.dgrad_splits, &q.dgrad_sps, q.G);
    // tail splits where the grid is not split already
    const int tail_forced = env_tile("CAFFE_CONV_TAIL_SPLITS");
    const int tail_cus = env_tile("CAFFE_CONV_TAIL_UNITS");
    q.fwd_tail = ConvPlan::Tail{0, 1, 0, 0, 0};
    q.dgrad_tail = ConvPlan::Tail{0, 1, 0, 0, 0};
    if (q.fwd_splits == 1)
        plan_tail(q.Kg, (int64_t)q.N * q.Ho * q.Wo, q.R, q.fwd_tile, q.G, cus, tail_forced,
                  tail_cus, &q.fwd_tail);
    if (q.dgrad_splits == 1)
        plan_tail(q.Mt, dcols, q.Rt, q.dgrad_tile, q.G, cus, tail_forced, tail_cus,
                  &q.dgrad_tail);
    const int64_t fpart = q.fwd_splits > 1 ? (int64_t)q.fwd_splits * q.top_elems * 4
                                           : q.fwd_tail.bytes;
    const int64_t dpart = q.dgrad_splits > 1
                              ? (int64_t)q.dgrad_splits * q.G * q.Mt * dcols * 4
                              : q.dgrad_tail.bytes;
    if (fpart > kMaxTensorBytes || dpart > kMaxTensorBytes)
        return fail(CAFFE_ERR_UNSUPPORTED, "split partials reach 2^31 bytes");
    q.off_fwd_part = q.ws_fwd;
    q.ws_fwd += align_up(fpart, kWsAlign);
    // channel-major forward gather: a tap-offset table (the kernel adds its
    // entries to lane offsets of up to X's size, hence the 2^30 bound)
    q.fwd_taps = !q.fwd_tap && q.bottom_elems * q.esize < (int64_t(1) << 30) &&
                 env_tile("CAFFE_CONV_TAP_TABLE") != 0;
    q.fwd_rpad = round_up(q.R, gemm_tile_k(q.fwd_tile));
    q.off_taps_fwd = q.ws_fwd;
    if (q.fwd_taps)
        q.ws_fwd += align_up((size_t)q.fwd_rpad * 4, kWsAlign);

    // Workspace: [masked top diff][bias partial sums][transformed weights]
    // [weight or data-gradient partials].  The masked top diff is written
    // only when relu is set and the caller has not masked top_diff already.
    const size_t d_bytes = q.relu ? align_up(q.top_elems * 4, kWsAlign) : 0;
    const size_t sums_bytes =
        align_up((size_t)std::max<int64_t>(q.N, q.splits) * q.K * 4, kWsAlign);
    const size_t wt_bytes = align_up(wt_elems * 4, kWsAlign);
    q.off_d = 0;
    q.off_sums = d_bytes;
    q.off_wt = q.off_sums + sums_bytes;
    q.off_part = q.off_wt + wt_bytes;
    q.ws_data = q.off_part + align_up(dpart, kWsAlign);
    q.off_coltab = q.off_part + align_up(part_bytes, kWsAlign);
    q.ws_weights = q.off_coltab + (q.wgrad_quad ? align_up((size_t)q.ncol_pad * 12, kWsAlign) : 0);
    q.ws_both = std::max(q.ws_data, q.ws_weights);
    return CAFFE_OK;
}

int check_ptr(const void* ptr, bool required, const char* name)
{
    if (!ptr) {
        if (required)
            return fail(CAFFE_ERR_INVALID_ARG, "%s is NULL", name);
        return CAFFE_OK;
    }
    if (!aligned(ptr, 16))
        return fail(CAFFE_ERR_ALIGN, "%s is not 16-byte aligned", name);
    return CAFFE_OK;
}

int check_ws(const void* ws, size_t ws_bytes, size_t need)
{
    if (need == 0)
        return CAFFE_OK;
    if (ws_bytes < need)
        return fail(CAFFE_ERR_WORKSPACE, "workspace of %zu bytes is smaller than the %zu needed",
                    ws_bytes, need);
    if (!ws)
        return fail(CAFFE_ERR_INVALID_ARG, "workspace is NULL");
    if (!aligned(ws, kWsAlign))
        return fail(CAFFE_ERR_ALIGN, "workspace is not 256-byte aligned");
    return CAFFE_OK;
}

#define CHECK(expr)                                                                               \
    do {                                                                                          \
        int _st = (expr);                                                                         \
        if (_st != CAFFE_OK)                                                                      \
            return _st;                                                                           \
    } while (0)

#define LAUNCH(expr, what)                                                                        \
    do {                                                                                          \
        hipError_t _e = (expr);                                                                   \
        if (_e != hipSuccess)                                                                     \
            return hip_fail(_e, what);                                                            \
    } while (0)

uint32_t nbytes(int64_t elems, int64_t esize) { return (uint32_t)(elems * esize); }

int run_forward(const ConvPlan& q, const void* bottom, const void* weight, const float* bias,
                float* top, char* ws, hipStream_t s)
{
    if (q.top_elems == 0)
        return CAFFE_OK;
    // weights transposed to [group][r][m] in the kernel's reduction order
    float* wp = (float*)ws;
    LAUNCH(launch_pack_weights((const float*)weight, wp, q.G, q.Kg, q.Cg, q.kh * q.kw,
                               gemm_tile_k(q.fwd_tile), q.fwd_tap ? (q.blocked ? 1 : -1) : 0,
                               s),
           "weight pack launch");
    ConvGemmParams p = {};
    p.A = wp;
    p.X = bottom;
    p.Y = top;
    p.bias = bias;
    p.A_bytes = nbytes(q.weight_elems, q.esize);
    p.X_bytes = nbytes(q.bottom_elems, q.esize);
    p.Y_bytes = nbytes(q.top_elems, 4);
    p.N = q.N; p.Cin = q.C; p.IH = q.H; p.IW = q.W; p.Cin_g = q.Cg;
    p.kh = q.kh; p.kw = q.kw; p.sh = q.sh; p.sw = q.sw; p.ph = q.ph; p.pw = q.pw;
    p.OH = q.Ho; p.OW = q.Wo;
    p.M = q.Kg; p.R = q.R; p.G = q.G;
    p.Ncol = q.N * q.Ho * q.Wo;
    p.relu = q.relu;
    p.Cout = q.K; p.OutH = q.Ho; p.OutW = q.Wo;
    p.blocked = q.blocked;
    p.xcd_order = q.xcd_order;
    if (q.fwd_taps) {
        uint32_t* taps = (uint32_t*)(ws + q.off_taps_fwd);
        LAUNCH(launch_tap_table(taps, q.fwd_rpad, q.R, q.kh, q.kw, q.H * q.W, q.W, p.X_bytes, s),
               "tap table launch");
        p.taps = taps;
    }
    if (q.fwd_splits > 1) {
        float* part = (float*)(ws + q.off_fwd_part);
        ConvGemmParams pp = p;
        pp.Y = part;
        pp.Y_bytes = nbytes((int64_t)q.fwd_splits * q.top_elems, 4);
        pp.splits = q.fwd_splits;
        pp.stages_per_split = q.fwd_sps;
        LAUNCH(launch_conv_gemm_f32(pp, 3, q.fwd_tile, q.fwd_tap, s), "forward launch");
        LAUNCH(launch_conv_split_reduce_fwd(part, q.fwd_splits, p, top, s),
               "forward reduce launch");
        return CAFFE_OK;
    }
    if (q.fwd_tail.splits > 1) {
        float* part = (float*)(ws + q.off_fwd_part);
        p.tail_T = q.fwd_tail.T;
        p.tail_splits = q.fwd_tail.splits;
        p.tail_sps = q.fwd_tail.sps;
        p.tail_c0 = q.fwd_tail.c0;
        p.Pt = part;
        p.Pt_bytes = nbytes(q.fwd_tail.bytes, 1);
        LAUNCH(launch_conv_gemm_f32(p, 0, q.fwd_tile, q.fwd_tap, s), "forward launch");
        LAUNCH(launch_conv_split_reduce_fwd(part, q.fwd_tail.splits, p, top, s, q.G - 1,
                                            q.fwd_tail.c0),
               "forward tail reduce launch");
        return CAFFE_OK;
    }
    LAUNCH(launch_conv_gemm_f32(p, 0, q.fwd_tile, q.fwd_tap, s), "forward launch");
    return CAFFE_OK;
}

// Bias gradient without a weight gradient: per-(n, k) plane sums of the
// masked top gradient, reduced over n in order.
int run_bias_only(const ConvPlan& q, const float* top_diff, const float* top, bool masked,
                  float* bias_diff, int accumulate, char* ws, hipStream_t s)
{
    float* sums = (float*)(ws + q.off_sums);
    if (q.N > 0)
        LAUNCH(launch_relu_mask_bias(top_diff, top, nullptr, sums, q.N * q.K, q.Ho * q.Wo,
                                     q.relu && !masked, s),
               "bias launch");
    LAUNCH(launch_wgrad_reduce(nullptr, nullptr, 0, 0, sums, bias_diff, q.N, q.K, accumulate, s),
           "bias reduce launch");
    return CAFFE_OK;
}

int run_data(const ConvPlan& q, const float* dsrc, const float* bottom_mask, const void* weight,
             float* bottom_diff, char* ws, hipStream_t s)
{
    if (q.bottom_elems == 0)
        return CAFFE_OK;
    float* wt = (float*)(ws + q.off_wt);
    LAUNCH(launch_dgrad_weight_transform((const float*)weight, wt, q.G, q.Kg, q.Cg, q.kh, q.kw,
                                         q.sh, q.sw, q.Th, q.Tw,
                                         q.dgrad_tap ? (q.blocked ? gemm_tile_k(q.dgrad_tile) : -1)
                                                     : 0,
                                         s),
           "weight transform launch");
    ConvGemmParams p = {};
    p.A = wt;
    p.X = dsrc;
    p.Omask = bottom_mask;
    p.Y = bottom_diff;
    p.bias = nullptr;
    p.A_bytes = nbytes((int64_t)q.G * q.Mt * q.Rt, 4);
    p.X_bytes = nbytes(q.top_elems, 4);
    p.Y_bytes = nbytes(q.bottom_elems, 4);
    p.N = q.N; p.Cin = q.K; p.IH = q.Ho; p.IW = q.Wo; p.Cin_g = q.Kg;
    p.kh = q.Th; p.kw = q.Tw; p.sh = 1; p.sw = 1;
    p.ph = q.Th - 1 - q.a0h; p.pw = q.Tw - 1 - q.a0w;  // may be negative: bounds-checked gather
    p.OH = q.Ah; p.OW = q.Aw;
    p.M = q.Mt; p.R = q.Rt; p.G = q.G;
    p.Ncol = q.N * q.Ah * q.Aw;
    p.relu = 0;
    p.Cout = q.C; p.OutH = q.H; p.OutW = q.W;
    p.psh = q.sh; p.psw = q.sw; p.a0h = q.a0h; p.a0w = q.a0w; p.oph = q.ph; p.opw = q.pw;
    p.Cg_out = q.Cg;
    p.blocked = q.blocked;
    p.xcd_order = q.xcd_order;
    p.div_pss = make_fastdiv((uint32_t)(q.sh * q.sw)); p.div_psw = make_fastdiv((uint32_t)q.sw);
    if (q.dgrad_splits > 1) {
        float* part = (float*)(ws + q.off_part);
        ConvGemmParams pp = p;
        pp.Y = part;
        pp.Y_bytes = nbytes((int64_t)q.dgrad_splits * q.G * q.Mt * p.Ncol, 4);
        pp.Omask = nullptr;
        pp.splits = q.dgrad_splits;
        pp.stages_per_split = q.dgrad_sps;
        LAUNCH(launch_conv_gemm_f32(pp, 3, q.dgrad_tile, q.dgrad_tap, s),
               "data-gradient launch");
        LAUNCH(launch_conv_split_reduce_dgrad(part, q.dgrad_splits, p, bottom_mask, bottom_diff,
                                              s),
               "data-gradient reduce launch");
        return CAFFE_OK;
    }
    if (q.dgrad_tail.splits > 1) {
        float* part = (float*)(ws + q.off_part);
        p.tail_T = q.dgrad_tail.T;
        p.tail_splits = q.dgrad_tail.splits;
        p.tail_sps = q.dgrad_tail.sps;
        p.tail_c0 = q.dgrad_tail.c0;
        p.Pt = part;
        p.Pt_bytes = nbytes(q.dgrad_tail.bytes, 1);
        LAUNCH(launch_conv_gemm_f32(p, 1, q.dgrad_tile, q.dgrad_tap, s),
               "data-gradient launch");
        LAUNCH(launch_conv_split_reduce_dgrad(part, q.dgrad_tail.splits, p, bottom_mask,
                                              bottom_diff, s, q.G - 1, q.dgrad_tail.c0),
               "data-gradient tail reduce launch");
        return CAFFE_OK;
    }
    LAUNCH(launch_conv_gemm_f32(p, 1, q.dgrad_tile, q.dgrad_tap, s), "data-gradient launch");
    return CAFFE_OK;
}

int run_weights(const ConvPlan& q, const float* dsrc, const void* bottom, float* weight_diff,
                float* bias_diff, int accumulate, char* ws, hipStream_t s)
{
    float* part = (float*)(ws + q.off_part);
    float* sums = (float*)(ws + q.off_sums);
    WgradParams p = {};
    p.D = dsrc;
    p.X = bottom;
    p.P = part;
    p.dbp = bias_diff ? sums : nullptr;
    p.D_bytes = nbytes(q.top_elems, 4);
    p.X_bytes = nbytes(q.bottom_elems, q.esize);
    p.P_bytes = nbytes((int64_t)q.splits * q.weight_elems, 4);
    p.N = q.N; p.C = q.C; p.IH = q.H; p.IW = q.W; p.Cg = q.Cg; p.K = q.K; p.Kg = q.Kg;
    p.kh = q.kh; p.kw = q.kw; p.sh = q.sh; p.sw = q.sw; p.ph = q.ph; p.pw = q.pw;
    p.OH = q.Ho; p.OW = q.Wo;
    p.R = q.R; p.G = q.G;
    p.Ncol = q.N * q.Ho * q.Wo;
    p.cols_per_split = q.cols_per_split;
    p.splits = q.splits;
    p.div_ohw = make_fastdiv((uint32_t)(q.Ho * q.Wo));
    p.div_ow = make_fastdiv((uint32_t)q.Wo);
    p.xcd_order = q.wgrad_xcd_order;
    p.unit_order = q.wgrad_unit_order ? 1 : 0;
    if (q.wgrad_quad) {
        uint32_t* tab = (uint32_t*)(ws + q.off_coltab);
        LAUNCH(launch_wgrad_col_table(tab, (int)p.Ncol, q.ncol_pad, q.C, q.H, q.W, q.K, q.Ho,
                                      q.Wo, q.kh, q.kw, q.sh, q.sw, q.ph, q.pw, s),
               "weight-gradient column table launch");
        p.T = tab;
        p.T_bytes = nbytes((int64_t)q.ncol_pad * 3, 4);
        p.xpad = q.xpad;
        if (q.wgrad_dma)
            LAUNCH(launch_conv_wgrad_dma_f32(p, q.wgrad_tile, s), "weight-gradient launch");
        else
            LAUNCH(launch_conv_wgrad_quad_f32(p, q.wgrad_tile, s), "weight-gradient launch");
    } else {
        LAUNCH(launch_conv_wgrad_f32(p, q.wgrad_tile, s), "weight-gradient launch");
    }
    // dW = sum of the split partials; db = sum of the split bias partials
    LAUNCH(launch_wgrad_reduce(part, weight_diff, (int)q.weight_elems, q.splits, sums, bias_diff,
                               q.splits, q.K, accumulate, s),
           "reduce launch");
    return CAFFE_OK;
}

// ---- inner product (dense split-K GEMMs)
ConvGemmParams dense_params(const float* A, uint32_t A_bytes, const float* X, uint32_t X_bytes,
                            float* P, uint32_t P_bytes, int M, int ncol, int R, int splits,
                            int sps)
{
    ConvGemmParams p = {};
    p.A = A;
    p.X = X;
    p.Y = P;
    p.A_bytes = A_bytes;
    p.X_bytes = X_bytes;
    p.Y_bytes = P_bytes;
    p.M = M;
    p.R = R;
    p.G = 1;
    p.Ncol = ncol;
    p.splits = splits;
    p.stages_per_split = sps;
    p.xcd_order = 1;
    return p;
}

int run_dense_forward(const ConvPlan& q, const float* bottom, const float* weight,
                      const float* bias, float* top, char* ws, hipStream_t s)
{
    const int N = q.N, C = q.C, K = q.K;
    if (N == 0)
        return CAFFE_OK;
    float* part = (float*)(ws + q.fc_off_pf);
    if (C % 4 == 0) {
        // both operands as stored: X [N][C] and W [K][C], C contiguous (and
        // 16-byte aligned, as every tensor argument)
        const ConvGemmParams p =
            dense_params(bottom, nbytes((int64_t)N * C, 4), weight, nbytes((int64_t)K * C, 4), part,
                         nbytes((int64_t)q.fc_splits_f * N * K, 4), N, K, C, q.fc_splits_f,
                         q.fc_sps_f);
        LAUNCH(launch_dense_gemm_nt_f32(p, q.fc_tile_f, s), "inner-product forward launch");
        LAUNCH(launch_split_reduce(part, q.fc_splits_f, N * K, K, bias, q.relu, nullptr, top, s),
               "inner-product reduce launch");
        return CAFFE_OK;
    }
    // otherwise through X^T [C][N] and W^T [C][K]
    float* xt = (float*)(ws + q.fc_off_xt);
    float* wp = (float*)(ws + q.fc_off_wp);
    LAUNCH(launch_transpose_f32(bottom, xt, N, C, s), "transpose launch");
    LAUNCH(launch_transpose_f32(weight, wp, K, C, s), "transpose launch");
    const ConvGemmParams p =
        dense_params(xt, nbytes((int64_t)N * C, 4), wp, nbytes((int64_t)K * C, 4), part,
                     nbytes((int64_t)q.fc_splits_f * N * K, 4), N, K, C, q.fc_splits_f,
                     q.fc_sps_f);
    LAUNCH(launch_dense_gemm_f32(p, q.fc_tile_f, s), "inner-product forward launch");
    LAUNCH(launch_split_reduce(part, q.fc_splits_f, N * K, K, bias, q.relu, nullptr, top, s),
           "inner-product reduce launch");
    return CAFFE_OK;
}

int backward_dense(const ConvPlan& q, const float* top_diff, const float* top, bool masked,
                   bool mask_bottom, const float* bottom, const float* weight, float* bottom_diff,
                   float* weight_diff, float* bias_diff, int accumulate, char* ws, hipStream_t s)
{
    const int N = q.N, C = q.C, K = q.K;
    const float* D = top_diff;
    if (q.relu && !masked && N > 0) {
        float* d = (float*)(ws + q.fc_off_d);
        LAUNCH(launch_relu_mask(top_diff, top, d, (int64_t)N * K, s), "ReLU backward launch");
        D = d;
    }
    float* part = (float*)(ws + q.fc_off_pb);
    if (bottom_diff && N > 0) {
        float* dt = (float*)(ws + q.fc_off_dt);
        LAUNCH(launch_transpose_f32(D, dt, N, K, s), "transpose launch");
        const ConvGemmParams p =
            dense_params(dt, nbytes((int64_t)N * K, 4), weight, nbytes((int64_t)K * C, 4), part,
                         nbytes((int64_t)q.fc_splits_d * N * C, 4), N, C, K, q.fc_splits_d,
                         q.fc_sps_d);
        LAUNCH(launch_dense_gemm_f32(p, q.fc_tile_d, s), "inner-product data-gradient launch");
        LAUNCH(launch_split_reduce(part, q.fc_splits_d, N * C, C, nullptr, 0,
                                   mask_bottom ? bottom : nullptr, bottom_diff, s),
               "inner-product reduce launch");
    }
    if (weight_diff) {
        // one split and no accumulation: the GEMM writes dW itself
        const bool direct = q.fc_splits_w == 1 && !accumulate;
        float* dst = direct ? weight_diff : part;
        if (N > 0) {
            const ConvGemmParams p =
                dense_params(D, nbytes((int64_t)N * K, 4), bottom, nbytes((int64_t)N * C, 4), dst,
                             nbytes((int64_t)q.fc_splits_w * K * C, 4), K, C, N, q.fc_splits_w,
                             q.fc_sps_w);
            LAUNCH(launch_dense_gemm_f32(p, q.fc_tile_w, s), "inner-product weight-gradient launch");
        } else if (!accumulate) {
            LAUNCH(launch_fill_zero(weight_diff, (int64_t)K * C, s), "zero fill launch");
        }
        // dW = sum of the split partials; db[k] = sum_n D[n][k]
        const bool sum_w = !direct && N > 0;
        LAUNCH(launch_wgrad_reduce(part, weight_diff, sum_w ? K * C : 0, q.fc_splits_w, D,
                                   bias_diff, N, K, accumulate, s),
               "reduce launch");
    } else if (bias_diff) {
        LAUNCH(launch_wgrad_reduce(nullptr, nullptr, 0, 0, D, bias_diff, N, K, accumulate, s),
               "bias reduce launch");
    }
    return CAFFE_OK;
}

// ---- bf16 operands
// The input's bf16 staging (plain or space-to-depth) at xh.
// Whether the LRN forward can write convolution qn's bf16 bottom staging:
// the plain channel-contiguous layout with unpadded groups, in whole
// 16-channel chunks.
bool caffe_hip_stage_from_lrn_ok(const ConvPlan& qn, int lrn_size)
{
    return is_bf16(qn) && !qn.s2d && qn.Cgp == qn.Cg && qn.C % 16 == 0 &&
           (lrn_size == 3 || lrn_size == 5) && qn.ph >= 0 && qn.pw >= 0;
}

hipError_t stage_bottom_bf16(const ConvPlan& q, const void* bottom, uint16_t* xh, hipStream_t s)
{
    if (q.s2d)
        return launch_stage_s2d_bf16(bottom, bottom_f32(q), xh, q.N, q.C, q.H, q.W, q.s2d, q.ph,
                                     q.pw, q.XHp, q.XWp, q.Cgp, s);
    return launch_stage_nhwc_bf16(bottom, bottom_f32(q), xh, q.N, q.C, q.H, q.W, q.Cg, q.Cgp,
                                  q.G * q.Cgp, q.XHp, q.XWp, q.ph, q.pw, s);
}

int run_forward_bf16(const ConvPlan& q, const void* bottom, const void* weight, const float* bias,
                     float* top, char* ws, hipStream_t s, bool bottom_staged = false)
{
    if (q.top_elems == 0)
        return CAFFE_OK;
    uint16_t* xh = (uint16_t*)(ws + q.off_xh_fwd);
    uint16_t* wp = (uint16_t*)(ws + q.off_wp_fwd);
    const int Ctot = q.G * q.Cgp;
    if (!bottom_staged)
        LAUNCH(stage_bottom_bf16(q, bottom, xh, s), "bf16 staging launch");
    LAUNCH(launch_pack_weights_bf16((const uint16_t*)weight, wp, q.K, q.Cg, q.Cgp, q.kh, q.kw,
                                    q.kwp, q.s2d ? q.s2d : 1, q.Rp, s),
           "bf16 weight pack launch");
    GemmBf16Params p = {};
    p.A = wp;
    p.X = xh;
    p.Y = top;
    p.bias = bias;
    p.A_bytes = nbytes((int64_t)q.K * q.Rp, 2);
    p.X_bytes = nbytes((int64_t)q.N * q.XHp * q.XWp * Ctot, 2);
    p.Y_bytes = nbytes(q.top_elems, 4);
    p.N = q.N; p.IHp = q.XHp; p.IWp = q.XWp; p.Ctot = Ctot; p.Cgp = q.Cgp;
    // chunks per tap group, tap groups per kernel row, elements per tap group
    p.Cg8 = q.Cgp >= 8 ? q.Cgp / 8 : 1;
    p.kw = q.kwp / q.tpc;
    p.vstr = q.Cgp >= 8 ? Ctot : 8;
    p.KC = q.gkh * p.kw * p.Cg8;
    p.div_cg8 = make_fastdiv((uint32_t)p.Cg8); p.div_kw = make_fastdiv((uint32_t)p.kw);
    p.kh = q.gkh; p.oh0 = 0; p.ow0 = 0;
    p.sh = q.s2d ? 1 : q.sh;
    p.sw = q.s2d ? 1 : q.sw;
    p.OH = q.Ho; p.OW = q.Wo;
    p.M = q.Kg; p.Rp = q.Rp; p.G = q.G;
    p.Ncol = q.N * q.Ho * q.Wo;
    p.relu = q.relu;
    p.Cout = q.K; p.OutH = q.Ho; p.OutW = q.Wo;
    p.xcd_order = q.xcd_order;
    p.div_ohw = make_fastdiv((uint32_t)(q.Ho * q.Wo)); p.div_ow = make_fastdiv((uint32_t)q.Wo);
    p.div_pss = make_fastdiv(1); p.div_psw = make_fastdiv(1);
    LAUNCH(launch_conv_gemm_bf16(p, 0, q.fwd_tile, q.fwd_pipe, s), "bf16 forward launch");
    return CAFFE_OK;
}

int run_data_bf16(const ConvPlan& q, const uint16_t* dh, const void* bottom_mask,
                  const void* weight, float* bottom_diff, char* ws, hipStream_t s)
{
    if (q.bottom_elems == 0)
        return CAFFE_OK;
    if (q.below)  // its border first (the epilogue writes the image's pixels)
        LAUNCH(launch_dh_zero_border(q.below->Sh, q.N, q.below->Hp, q.below->Wp, q.below->tb,
                                     q.below->lb, q.H, q.W, q.below->Ktot, s),
               "staging border launch");
    uint16_t* wt = (uint16_t*)(ws + q.off_wt);
    LAUNCH(launch_dgrad_weights_bf16((const uint16_t*)weight, wt, q.G, q.Kg, q.Kgp, q.Cg, q.kh,
                                     q.kw, q.sh, q.sw, q.Th, q.Tw, q.Rtp, q.dgrad_blocked, s),
           "bf16 weight transform launch");
    const int Ktot = q.G * q.Kgp;
    GemmBf16Params p = {};
    p.A = wt;
    p.X = dh;
    p.Omask = bottom_mask;
    p.omask_f32 = bottom_f32(q);
    p.Y = bottom_diff;
    p.A_bytes = nbytes((int64_t)q.G * q.Mt * q.Rtp, 2);
    p.X_bytes = nbytes((int64_t)q.N * q.DHp * q.DWp * Ktot, 2);
    p.Y_bytes = nbytes(q.bottom_elems, 4);
    p.N = q.N; p.IHp = q.DHp; p.IWp = q.DWp; p.Ctot = Ktot; p.Cgp = q.Kgp;
    p.Cg8 = q.Kgp / 8; p.KC = q.Th * q.Tw * p.Cg8; p.vstr = Ktot;
    p.div_cg8 = make_fastdiv((uint32_t)p.Cg8); p.div_kw = make_fastdiv((uint32_t)q.Tw);
    p.kh = q.Th; p.kw = q.Tw; p.sh = 1; p.sw = 1; p.oh0 = q.doh0; p.ow0 = q.dow0;
    p.OH = q.Ah; p.OW = q.Aw;
    p.M = q.Mt; p.Rp = q.Rtp; p.G = q.G;
    p.Ncol = q.N * q.Ah * q.Aw;
    p.Cout = q.C; p.OutH = q.H; p.OutW = q.W;
    p.psh = q.sh; p.psw = q.sw; p.a0h = q.a0h; p.a0w = q.a0w; p.oph = q.ph; p.opw = q.pw;
    p.Cg_out = q.Cg;
    p.xcd_order = q.xcd_order;
    p.blocked = q.dgrad_blocked;
    p.ntap = q.Th * q.Tw;
    p.div_ntap = make_fastdiv((uint32_t)p.ntap);
    p.div_ohw = make_fastdiv((uint32_t)(q.Ah * q.Aw)); p.div_ow = make_fastdiv((uint32_t)q.Aw);
    p.div_pss = make_fastdiv((uint32_t)(q.sh * q.sw)); p.div_psw = make_fastdiv((uint32_t)q.sw);
    if (q.below) {
        const ConvPlan::StageTarget& b = *q.below;
        p.Y = nullptr;
        p.Sh = b.Sh; p.Ssum = b.Ssum; p.Sh_bytes = b.Sh_bytes; p.Ssum_bytes = b.Ssum_bytes;
        p.s_Hp = b.Hp; p.s_Wp = b.Wp; p.s_tb = b.tb; p.s_lb = b.lb; p.s_Ktot = b.Ktot;
        p.s_T = b.T;
        LAUNCH(launch_conv_gemm_bf16(p, 2, q.dgrad_tile, q.dgrad_pipe, s),
               "bf16 data-gradient staging launch");
        return CAFFE_OK;
    }
    LAUNCH(launch_conv_gemm_bf16(p, 1, q.dgrad_tile, q.dgrad_pipe, s),
           "bf16 data-gradient launch");
    return CAFFE_OK;
}

int run_weights_bf16(const ConvPlan& q, const uint16_t* dh, const void* bottom, bool staged,
                     float* weight_diff, int accumulate, char* ws, hipStream_t s)
{
    uint16_t* xh = (uint16_t*)(ws + q.off_xh);
    float* part = (float*)(ws + q.off_part);
    const int Ctot = q.G * q.Cgp;
    if (!staged)
        LAUNCH(stage_bottom_bf16(q, bottom, xh, s), "bf16 staging launch");
    WgradBf16Params p = {};
    p.D = dh;
    p.X = xh;
    p.P = part;
    p.D_bytes = nbytes((int64_t)q.N * q.DHp * q.DWp * q.G * q.Kgp, 2);
    p.X_bytes = nbytes((int64_t)q.N * q.XHp * q.XWp * Ctot, 2);
    p.P_bytes = nbytes((int64_t)q.splits * q.K * q.Rw, 4);
    p.N = q.N; p.IHp = q.XHp; p.IWp = q.XWp; p.Ctot = Ctot; p.Cgp = q.Cgp;
    p.K = q.K; p.Kg = q.Kg; p.Kgp = q.Kgp; p.Ktot = q.G * q.Kgp;
    p.DHp = q.DHp; p.DWp = q.DWp; p.dtb = q.dtb; p.dlb = q.dlb;
    p.kh = q.gkh; p.kw = q.kwp;
    p.sh = q.s2d ? 1 : q.sh;
    p.sw = q.s2d ? 1 : q.sw;
    p.OH = q.Ho; p.OW = q.Wo;
    p.Rw = q.Rw; p.G = q.G;
    p.Ncol = q.N * q.Ho * q.Wo;
    p.cols_per_split = q.cols_per_split;
    p.splits = q.splits;
    p.div_ohw = make_fastdiv((uint32_t)(q.Ho * q.Wo));
    p.div_ow = make_fastdiv((uint32_t)q.Wo);
    p.unit_order = q.wgrad_unit_order ? 1 : 0;
    LAUNCH(launch_conv_wgrad_bf16(p, q.wgrad_tile, s), "bf16 weight-gradient launch");
    LAUNCH(launch_wgrad_reduce_perm(part, weight_diff, q.K, q.Rw, q.Cgp, q.Cg, q.kh, q.kw, q.kwp,
                                    q.s2d ? q.s2d : 1, q.splits, accumulate, s),
           "bf16 reduce launch");
    return CAFFE_OK;
}

// A combined bf16 backward call with both gradients runs the weight gradient
// on a second stream of the device (created once, default priority), forked
// after the shared top-gradient staging and joined before the call returns:
// the two GEMMs fill each other's idle compute units (the CaffeNet bf16
// step at N=512: 5.35 -> 5.29 ms; the fp32 path measured no gain).  Not under
// graph capture, and not when CAFFE_BACKWARD_FORK=0.
hipStream_t device_side_stream()
{
    static std::mutex mu;
    static hipStream_t streams[64] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64)
        return nullptr;
    std::lock_guard<std::mutex> lock(mu);
    if (!streams[dev] && hipStreamCreateWithFlags(&streams[dev], hipStreamNonBlocking) != hipSuccess)
        streams[dev] = nullptr;
    return streams[dev];
}

struct Fork {
    hipStream_t side = nullptr;
    hipEvent_t start = nullptr, done = nullptr;
};

// true: work enqueued on f->side after this call follows everything enqueued
// on s so far
bool fork_side(hipStream_t s, Fork* f)
{
    if (env_tile("CAFFE_BACKWARD_FORK") == 0)
        return false;
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(s, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone)
        return false;
    f->side = device_side_stream();
    if (!f->side)
        return false;
    if (hipEventCreateWithFlags(&f->start, hipEventDisableTiming) != hipSuccess)
        return false;
    if (hipEventCreateWithFlags(&f->done, hipEventDisableTiming) != hipSuccess ||
        hipEventRecord(f->start, s) != hipSuccess ||
        hipStreamWaitEvent(f->side, f->start, 0) != hipSuccess) {
        (void)hipEventDestroy(f->start);
        if (f->done)
            (void)hipEventDestroy(f->done);
        return false;
    }
    return true;
}

// s then follows everything enqueued on f.side; st_a / st_b: the two
// branches' statuses (the first failure is returned)
int join_side(hipStream_t s, Fork& f, int st_a, int st_b)
{
    const hipError_t e1 = hipEventRecord(f.done, f.side);
    const hipError_t e2 = e1 == hipSuccess ? hipStreamWaitEvent(s, f.done, 0) : e1;
    if (e2 != hipSuccess) {
        // s cannot be made to wait for the side stream: drain the side stream
        // here, so that no kernel of this call still reads or writes the
        // caller's buffers or workspace once the error is returned
        (void)hipStreamSynchronize(f.side);
    }
    (void)hipEventDestroy(f.start);
    (void)hipEventDestroy(f.done);
    if (st_a != CAFFE_OK)
        return st_a;
    if (st_b != CAFFE_OK)
        return st_b;
    if (e2 != hipSuccess)
        return hip_fail(e2, "stream join");
    return CAFFE_OK;
}

// Work enqueued on `follower` after this call follows everything enqueued on
// `s` so far.
int stream_follow(hipStream_t follower, hipStream_t s)
{
    hipEvent_t ev = nullptr;
    hipError_t e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
    if (e == hipSuccess) {
        e = hipEventRecord(ev, s);
        if (e == hipSuccess)
            e = hipStreamWaitEvent(follower, ev, 0);
        (void)hipEventDestroy(ev);
    }
    if (e != hipSuccess)
        return hip_fail(e, "stream ordering");
    return CAFFE_OK;
}

int backward_bf16_staged(const ConvPlan& q, const float* sums, int terms, bool mask_bottom,
                         bool staged, const void* bottom, const void* weight, float* bottom_diff,
                         float* weight_diff, float* bias_diff, int accumulate, char* ws,
                         hipStream_t s, hipStream_t wst);

int backward_bf16(const ConvPlan& q, const float* top_diff, const float* top, bool masked,
                  bool top_staged, bool mask_bottom, bool staged, const void* bottom,
                  const void* weight, float* bottom_diff, float* weight_diff, float* bias_diff,
                  int accumulate, char* ws, hipStream_t s, hipStream_t wst)
{
    float* sums = (float*)(ws + q.off_sums);
    // the top gradient and its bias partials staged by the layer above
    const int staged_terms = stage_below_terms((int64_t)q.N * q.Ho * q.Wo);
    if (!bottom_diff && !weight_diff && !q.below) {
        if (bias_diff && top_staged)
            LAUNCH(launch_bias_reduce(sums, bias_diff, staged_terms, q.K, accumulate, s),
                   "bias reduce launch");
        else if (bias_diff)
            CHECK(run_bias_only(q, top_diff, top, masked, bias_diff, accumulate, ws, s));
        return wst ? stream_follow(wst, s) : CAFFE_OK;
    }
    if (top_staged)
        return backward_bf16_staged(q, sums, staged_terms, mask_bottom, staged, bottom, weight,
                                    bottom_diff, weight_diff, bias_diff, accumulate, ws, s, wst);
    uint16_t* dh = (uint16_t*)(ws + q.off_dh);
    // D = bf16(top_diff [top > 0]) staged channel-contiguous; the fp32 plane
    // sums give the bias gradient
    LAUNCH(launch_diff_prep_bf16(top_diff, top, dh, bias_diff ? sums : nullptr, q.N, q.K, q.Ho,
                                 q.Wo, q.Kg, q.Kgp, q.G * q.Kgp, q.DHp, q.DWp, q.dtb, q.dlb,
                                 q.relu && !masked, s),
           "bf16 top-gradient staging launch");
    return backward_bf16_staged(q, sums, diff_prep_terms(q.N, q.DHp * q.DWp), mask_bottom, staged,
                                bottom, weight, bottom_diff, weight_diff, bias_diff, accumulate, ws,
                                s, wst);
}

// The bf16 backward once the top gradient is staged at off_dh and its
// bias-gradient partials sit in `sums` (`terms` per channel).
int backward_bf16_staged(const ConvPlan& q, const float* sums, int terms, bool mask_bottom,
                         bool staged, const void* bottom, const void* weight, float* bottom_diff,
                         float* weight_diff, float* bias_diff, int accumulate, char* ws,
                         hipStream_t s, hipStream_t wst)
{
    const uint16_t* dh = (const uint16_t*)(ws + q.off_dh);
    const bool want_data = bottom_diff || q.below;
    if (wst) {
        // the caller's weight stream takes the weight and bias gradients
        // once the staging on s is done, and nothing joins it here (the two
        // passes use disjoint workspace regions, as in the fork below)
        CHECK(stream_follow(wst, s));
        if (want_data)
            CHECK(run_data_bf16(q, dh, mask_bottom ? bottom : nullptr, weight, bottom_diff, ws,
                                s));
        if (weight_diff)
            CHECK(run_weights_bf16(q, dh, bottom, staged, weight_diff, accumulate, ws, wst));
        if (bias_diff)
            LAUNCH(launch_bias_reduce(sums, bias_diff, terms, q.K, accumulate, wst),
                   "bias reduce launch");
        return CAFFE_OK;
    }
    Fork f;
    if (want_data && weight_diff && fork_side(s, &f)) {
        // (disjoint workspace regions: Wt for the data gradient; the staged
        // bottom and the partials for the weight gradient)
        const int sw = run_weights_bf16(q, dh, bottom, staged, weight_diff, accumulate, ws, f.side);
        const int sd =
            run_data_bf16(q, dh, mask_bottom ? bottom : nullptr, weight, bottom_diff, ws, s);
        CHECK(join_side(s, f, sw, sd));
    } else {
        if (want_data)
            CHECK(run_data_bf16(q, dh, mask_bottom ? bottom : nullptr, weight, bottom_diff, ws,
                                s));
        if (weight_diff)
            CHECK(run_weights_bf16(q, dh, bottom, staged, weight_diff, accumulate, ws, s));
    }
    if (bias_diff)
        LAUNCH(launch_bias_reduce(sums, bias_diff, terms, q.K, accumulate, s),
               "bias reduce launch");
    return CAFFE_OK;
}

// caffe_conv_backward_pool_lrn: the bf16 staging is written by the fused
// glue backward when a 16-channel block lies in one group; its bias partials
// (at most one per image, row strip and channel) go after the backward's
// workspace.  Otherwise the fp32 top gradient goes there.
bool pool_lrn_staged(const ConvPlan& q) { return is_bf16(q) && q.Kg % 16 == 0; }

size_t pool_lrn_extra(const ConvPlan& q)
{
    const int64_t elems = pool_lrn_staged(q) ? (int64_t)q.N * q.Ho * q.K : q.top_elems;
    return align_up((size_t)elems * 4, kWsAlign);
}

int check_conv_ptrs(const ConvPlan& q, const void* p, bool needed, bool is_blob, const char* name)
{
    // blob pointers may be NULL for an empty batch
    const bool required = needed && (!is_blob || q.N > 0);
    return check_ptr(p, required, name);
}

}  // namespace

extern "C" {

int caffe_conv_out_shape(const caffe_conv_desc* desc, int32_t* Ho, int32_t* Wo)
{
    ConvPlan q;
    CHECK(plan_conv(desc, &q));
    if (!Ho || !Wo)
        return fail(CAFFE_ERR_INVALID_ARG, "Ho/Wo is NULL");
    *Ho = q.Ho;
    *Wo = q.Wo;
    return CAFFE_OK;
}

int caffe_conv_workspace_size(const caffe_conv_desc* desc, int32_t pass, size_t* bytes)
{
    ConvPlan q;
    CHECK(plan_conv(desc, &q));
    if (!bytes)
        return fail(CAFFE_ERR_INVALID_ARG, "bytes is NULL");
    switch (pass) {
    case CAFFE_PASS_FORWARD:
        *bytes = q.ws_fwd;
        return CAFFE_OK;
    case CAFFE_PASS_BACKWARD_DATA:
        *bytes = q.ws_data;
        return CAFFE_OK;
    case CAFFE_PASS_BACKWARD_WEIGHTS:
        *bytes = q.ws_weights;
        return CAFFE_OK;
    case CAFFE_PASS_BACKWARD:
        *bytes = q.ws_both;
        return CAFFE_OK;
    case CAFFE_PASS_BACKWARD_POOL_LRN:
        *bytes = q.ws_both + pool_lrn_extra(q);
        return CAFFE_OK;
    default:
        return fail(CAFFE_ERR_INVALID_ARG, "unknown pass %d", pass);
    }
}

int caffe_conv_forward(const caffe_conv_desc* desc, const void* bottom, const void* weight,
                       const float* bias, float* top, void* workspace, size_t ws_bytes,
                       void* stream)
{
    return caffe_conv_forward_ex(desc, bottom, weight, bias, top, workspace, ws_bytes, 0, stream);
}

int caffe_conv_forward_ex(const caffe_conv_desc* desc, const void* bottom, const void* weight,
                          const float* bias, float* top, void* workspace, size_t ws_bytes,
                          int32_t flags, void* stream)
{
    ConvPlan q;
    CHECK(plan_conv(desc, &q));
    if (flags & ~CAFFE_FORWARD_BOTTOM_STAGED)
        return fail(CAFFE_ERR_INVALID_ARG, "unknown forward flags 0x%x", flags);
    const bool bottom_staged = (flags & CAFFE_FORWARD_BOTTOM_STAGED) != 0;
    if (bottom_staged && !is_bf16(q))
        return fail(CAFFE_ERR_INVALID_ARG, "CAFFE_FORWARD_BOTTOM_STAGED needs a bf16 mode");
    CHECK(check_conv_ptrs(q, bottom, !bottom_staged, true, "bottom"));
    CHECK(check_conv_ptrs(q, weight, true, false, "weight"));
    CHECK(check_conv_ptrs(q, bias, false, false, "bias"));
    CHECK(check_conv_ptrs(q, top, true, true, "top"));
    CHECK(check_ws(workspace, ws_bytes, q.ws_fwd));
    if (is_bf16(q))
        return run_forward_bf16(q, bottom, weight, bias, top, (char*)workspace,
                                (hipStream_t)stream, bottom_staged);
    if (q.dense)
        return run_dense_forward(q, (const float*)bottom, (const float*)weight, bias, top,
                                 (char*)workspace, (hipStream_t)stream);
    return run_forward(q, bottom, weight, bias, top, (char*)workspace, (hipStream_t)stream);
}

int caffe_conv_forward_noalloc(const caffe_conv_desc* desc, const void* bottom,
                               const void* weight, const float* bias, float* top, void* stream)
{
    static_assert(CAFFE_CONV_NOALLOC_SCRATCH_BYTES == caffe_hip::kStaticScratchBytes,
                  "header and library agree on the scratch size");
    ConvPlan q;
    CHECK(plan_conv(desc, &q));
    if (q.ws_fwd > caffe_hip::kStaticScratchBytes)
        return fail(CAFFE_ERR_WORKSPACE,
                    "the forward pass needs %zu bytes of workspace; the static scratch holds %zu",
                    q.ws_fwd, caffe_hip::kStaticScratchBytes);
    void* ws = nullptr;
    if (q.ws_fwd > 0) {
        const hipError_t e = caffe_hip::static_scratch_address(&ws);
        if (e != hipSuccess)
            return hip_fail(e, "static scratch lookup");
    }
    // the same checks and kernels as caffe_conv_forward, on the static buffer
    return caffe_conv_forward(desc, bottom, weight, bias, top, ws, q.ws_fwd, stream);
}

int caffe_conv_backward(const caffe_conv_desc* desc, const float* top_diff, const float* top,
                        const void* bottom, const void* weight, float* bottom_diff,
                        float* weight_diff, float* bias_diff, int32_t accumulate, int32_t flags,
                        void* workspace, size_t ws_bytes, void* stream)
{
    return caffe_conv_backward_ex(desc, top_diff, top, bottom, weight, bottom_diff, weight_diff,
                                  bias_diff, accumulate, flags, workspace, ws_bytes, stream,
                                  stream);
}

}  // extern "C"

namespace {

// Whether layer q's data gradient can be staged as the top gradient of the
// layer qb below it (see caffe_conv_backward_into): CAFFE_OK, else the error.
int check_stage_below(const ConvPlan& q, const ConvPlan& qb)
{
    if (!is_bf16(q) || !is_bf16(qb))
        return fail(CAFFE_ERR_UNSUPPORTED, "a staged data gradient needs bf16 modes");
    if (qb.N != q.N || qb.K != q.C || qb.Ho != q.H || qb.Wo != q.W)
        return fail(CAFFE_ERR_INVALID_ARG, "the layer below's top (%d, %d, %d, %d) is not this "
                    "layer's bottom (%d, %d, %d, %d)", qb.N, qb.K, qb.Ho, qb.Wo, q.N, q.C, q.H,
                    q.W);
    // stride 1 with the image as the GEMM's grid, no padded channels below
    if (q.sh != 1 || q.sw != 1 || q.Ah != q.H || q.Aw != q.W || q.a0h != q.ph ||
        q.a0w != q.pw || q.Cg % 4 != 0 || qb.Kgp != qb.Kg ||
        (q.dgrad_tile != BTILE_128x256 && q.dgrad_tile != BTILE_64x256))
        return fail(CAFFE_ERR_UNSUPPORTED, "this layer's data gradient cannot be staged for the "
                    "layer below (stride %dx%d, %d channels per group)", q.sh, q.sw, q.Cg);
    return CAFFE_OK;
}

// caffe_conv_backward_ex, and with `below` caffe_conv_backward_into (its
// data gradient staged into the layer below's workspace instead of stored).
int backward_impl(const caffe_conv_desc* desc, const float* top_diff, const float* top,
                  const void* bottom, const void* weight, float* bottom_diff, float* weight_diff,
                  float* bias_diff, int32_t accumulate, int32_t flags, void* workspace,
                  size_t ws_bytes, void* stream, void* weight_stream,
                  const caffe_conv_desc* below, void* below_ws, size_t below_ws_bytes)
{
    ConvPlan q;
    CHECK(plan_conv(desc, &q));
    if (accumulate != 0 && accumulate != 1)
        return fail(CAFFE_ERR_INVALID_ARG, "accumulate must be 0 or 1");
    if (flags & ~(CAFFE_BACKWARD_TOP_DIFF_MASKED | CAFFE_BACKWARD_MASK_BOTTOM_DIFF |
                  CAFFE_BACKWARD_BOTTOM_STAGED | CAFFE_BACKWARD_TOP_STAGED))
        return fail(CAFFE_ERR_INVALID_ARG, "unknown backward flags 0x%x", flags);
    const bool staged = (flags & CAFFE_BACKWARD_BOTTOM_STAGED) != 0;
    const bool top_staged = (flags & CAFFE_BACKWARD_TOP_STAGED) != 0;
    const bool masked = (flags & CAFFE_BACKWARD_TOP_DIFF_MASKED) != 0 || top_staged;
    if (top_staged && !is_bf16(q))
        return fail(CAFFE_ERR_INVALID_ARG, "CAFFE_BACKWARD_TOP_STAGED needs a bf16 mode");
    // the stage target: the layer below, whose top is this layer's bottom
    ConvPlan qb;
    ConvPlan::StageTarget target;
    if (below) {
        CHECK(plan_conv(below, &qb));
        CHECK(check_stage_below(q, qb));
        CHECK(check_ws(below_ws, below_ws_bytes, qb.ws_both));
        if (bottom_diff)
            return fail(CAFFE_ERR_INVALID_ARG, "bottom_diff is staged for the layer below: pass "
                        "NULL");
        target.Sh = (uint16_t*)((char*)below_ws + qb.off_dh);
        target.Ssum = (float*)((char*)below_ws + qb.off_sums);
        target.Hp = qb.DHp;
        target.Wp = qb.DWp;
        target.tb = qb.dtb;
        target.lb = qb.dlb;
        target.Ktot = qb.G * qb.Kgp;
        target.T = stage_below_terms((int64_t)qb.N * qb.Ho * qb.Wo);
        target.Sh_bytes = nbytes((int64_t)qb.N * qb.DHp * qb.DWp * target.Ktot, 2);
        target.Ssum_bytes = nbytes((int64_t)target.T * qb.K, 4);
        q.below = &target;
    }
    const bool want_dx = bottom_diff || below;
    const bool mask_bottom = (flags & CAFFE_BACKWARD_MASK_BOTTOM_DIFF) != 0 && want_dx;
    CHECK(check_conv_ptrs(q, top_diff, !top_staged, true, "top_diff"));
    CHECK(check_conv_ptrs(q, top, q.relu != 0 && !masked, true, "top"));
    CHECK(check_conv_ptrs(q, bottom, weight_diff != nullptr || mask_bottom, true, "bottom"));
    CHECK(check_conv_ptrs(q, weight, want_dx, false, "weight"));
    CHECK(check_conv_ptrs(q, bottom_diff, false, true, "bottom_diff"));
    CHECK(check_conv_ptrs(q, weight_diff, false, false, "weight_diff"));
    CHECK(check_conv_ptrs(q, bias_diff, false, false, "bias_diff"));
    // the pass sizes of caffe_conv_workspace_size: both gradients, data only,
    // weights (with or without the bias) only; the bias alone fits either
    const size_t need = want_dx && weight_diff ? q.ws_both
                        : want_dx              ? q.ws_data
                        : weight_diff          ? q.ws_weights
                                               : std::min(q.ws_data, q.ws_weights);
    CHECK(check_ws(workspace, ws_bytes, need));
    hipStream_t s = (hipStream_t)stream;
    // a weight stream other than `stream` takes the weight-side outputs
    hipStream_t wst = weight_stream != stream ? (hipStream_t)weight_stream : nullptr;
    char* ws = (char*)workspace;
    if (is_bf16(q))
        return backward_bf16(q, top_diff, top, masked, top_staged, mask_bottom, staged, bottom,
                             weight, bottom_diff, weight_diff, bias_diff, accumulate, ws, s, wst);
    if (q.dense) {
        CHECK(backward_dense(q, top_diff, top, masked, mask_bottom, (const float*)bottom,
                             (const float*)weight, bottom_diff, weight_diff, bias_diff,
                             accumulate, ws, s));
        return wst ? stream_follow(wst, s) : CAFFE_OK;
    }
    const float* dsrc = top_diff;
    if (q.relu && !masked && (bottom_diff || weight_diff) && q.top_elems > 0) {
        // D = top_diff [top > 0], shared by both gradients
        float* D = (float*)(ws + q.off_d);
        LAUNCH(launch_relu_mask_bias(top_diff, top, D, nullptr, q.N * q.K, q.Ho * q.Wo, 1, s),
               "ReLU backward launch");
        dsrc = D;
    }
    if (bottom_diff)
        CHECK(run_data(q, dsrc, mask_bottom ? (const float*)bottom : nullptr, weight, bottom_diff,
                       ws, s));
    if (weight_diff)
        CHECK(run_weights(q, dsrc, bottom, weight_diff, bias_diff, accumulate, ws, s));
    else if (bias_diff)
        CHECK(run_bias_only(q, top_diff, top, masked, bias_diff, accumulate, ws, s));
    // (fp32: both passes share the workspace's partial-sum region, so they
    // run in turn on `stream`)
    return wst ? stream_follow(wst, s) : CAFFE_OK;
}

}  // namespace

extern "C" {

int caffe_conv_backward_ex(const caffe_conv_desc* desc, const float* top_diff, const float* top,
                           const void* bottom, const void* weight, float* bottom_diff,
                           float* weight_diff, float* bias_diff, int32_t accumulate,
                           int32_t flags, void* workspace, size_t ws_bytes, void* stream,
                           void* weight_stream)
{
    return backward_impl(desc, top_diff, top, bottom, weight, bottom_diff, weight_diff, bias_diff,
                         accumulate, flags, workspace, ws_bytes, stream, weight_stream, nullptr,
                         nullptr, 0);
}

int caffe_conv_stage_below_supported(const caffe_conv_desc* desc, const caffe_conv_desc* below)
{
    ConvPlan q, qb;
    if (plan_conv(desc, &q) != CAFFE_OK || !below || plan_conv(below, &qb) != CAFFE_OK)
        return 0;
    return check_stage_below(q, qb) == CAFFE_OK ? 1 : 0;
}

int caffe_conv_backward_into(const caffe_conv_desc* desc, const float* top_diff, const float* top,
                             const void* bottom, const void* weight, float* weight_diff,
                             float* bias_diff, int32_t accumulate, int32_t flags,
                             void* workspace, size_t ws_bytes, const caffe_conv_desc* below,
                             void* below_workspace, size_t below_ws_bytes, void* stream,
                             void* weight_stream)
{
    if (!below)
        return fail(CAFFE_ERR_INVALID_ARG, "below is NULL");
    return backward_impl(desc, top_diff, top, bottom, weight, nullptr, weight_diff, bias_diff,
                         accumulate, flags, workspace, ws_bytes, stream, weight_stream, below,
                         below_workspace, below_ws_bytes);
}

int caffe_conv_backward_data(const caffe_conv_desc* desc, const float* top_diff, const float* top,
                             const void* weight, float* bottom_diff, void* workspace,
                             size_t ws_bytes, void* stream)
{
    ConvPlan q;
    CHECK(plan_conv(desc, &q));
    CHECK(check_conv_ptrs(q, bottom_diff, true, true, "bottom_diff"));
    return caffe_conv_backward(desc, top_diff, top, nullptr, weight, bottom_diff, nullptr, nullptr,
                               0, 0, workspace, ws_bytes, stream);
}

int caffe_conv_backward_weights(const caffe_conv_desc* desc, const float* top_diff,
                                const float* top, const void* bottom, float* weight_diff,
                                float* bias_diff, int32_t accumulate, void* workspace,
                                size_t ws_bytes, void* stream)
{
    ConvPlan q;
    CHECK(plan_conv(desc, &q));
    CHECK(check_conv_ptrs(q, weight_diff, true, false, "weight_diff"));
    return caffe_conv_backward(desc, top_diff, top, bottom, nullptr, nullptr, weight_diff,
                               bias_diff, accumulate, 0, workspace, ws_bytes, stream);
}

static int check_pool_lrn(const caffe_pool_desc* pd, const caffe_lrn_desc* ld, int* Ho, int* Wo);

int caffe_conv_backward_pool_lrn(const caffe_conv_desc* desc, const caffe_pool_desc* pool,
                                 const caffe_lrn_desc* lrn, const float* pooled,
                                 const float* lrn_top, const float* lrn_top_diff,
                                 const int32_t* pool_mask, const float* top, const void* bottom,
                                 const void* weight, float* bottom_diff, float* weight_diff,
                                 float* bias_diff, int32_t accumulate, int32_t flags,
                                 void* workspace, size_t ws_bytes, void* stream)
{
    return caffe_conv_backward_pool_lrn_ex(desc, pool, lrn, pooled, lrn_top, lrn_top_diff,
                                           pool_mask, top, bottom, weight, bottom_diff,
                                           weight_diff, bias_diff, accumulate, flags, workspace,
                                           ws_bytes, stream, stream);
}

int caffe_conv_backward_pool_lrn_ex(const caffe_conv_desc* desc, const caffe_pool_desc* pool,
                                    const caffe_lrn_desc* lrn, const float* pooled,
                                    const float* lrn_top, const float* lrn_top_diff,
                                    const int32_t* pool_mask, const float* top,
                                    const void* bottom, const void* weight, float* bottom_diff,
                                    float* weight_diff, float* bias_diff, int32_t accumulate,
                                    int32_t flags, void* workspace, size_t ws_bytes, void* stream,
                                    void* weight_stream)
{
    ConvPlan q;
    CHECK(plan_conv(desc, &q));
    int PHo, PWo;
    CHECK(check_pool_lrn(pool, lrn, &PHo, &PWo));
    if (pool->N != q.N || pool->C != q.K || pool->H != q.Ho || pool->W != q.Wo)
        return fail(CAFFE_ERR_INVALID_ARG, "the pooled blob (%d, %d, %d, %d) is not the "
                    "convolution's top (%d, %d, %d, %d)", pool->N, pool->C, pool->H, pool->W, q.N,
                    q.K, q.Ho, q.Wo);
    if (accumulate != 0 && accumulate != 1)
        return fail(CAFFE_ERR_INVALID_ARG, "accumulate must be 0 or 1");
    if (flags & ~(CAFFE_BACKWARD_TOP_DIFF_MASKED | CAFFE_BACKWARD_MASK_BOTTOM_DIFF |
                  CAFFE_BACKWARD_BOTTOM_STAGED | CAFFE_BACKWARD_POOL_MASK_OFFSETS))
        return fail(CAFFE_ERR_INVALID_ARG, "unknown backward flags 0x%x", flags);
    const int mask_u8 = (flags & CAFFE_BACKWARD_POOL_MASK_OFFSETS) ? 1 : 0;
    if (mask_u8 && pool->kernel_h * pool->kernel_w > 255)
        return fail(CAFFE_ERR_UNSUPPORTED, "byte winner offsets need windows of at most 255 taps");
    flags &= ~CAFFE_BACKWARD_POOL_MASK_OFFSETS;
    const bool masked = (flags & CAFFE_BACKWARD_TOP_DIFF_MASKED) != 0;
    const bool mask_bottom = (flags & CAFFE_BACKWARD_MASK_BOTTOM_DIFF) != 0 && bottom_diff;
    CHECK(check_conv_ptrs(q, pooled, true, true, "pooled"));
    CHECK(check_conv_ptrs(q, lrn_top, true, true, "lrn_top"));
    CHECK(check_conv_ptrs(q, lrn_top_diff, true, true, "lrn_top_diff"));
    CHECK(check_conv_ptrs(q, pool_mask, true, true, "pool_mask"));
    CHECK(check_conv_ptrs(q, top, q.relu != 0 && !masked, true, "top"));
    CHECK(check_conv_ptrs(q, bottom, weight_diff != nullptr || mask_bottom, true, "bottom"));
    CHECK(check_conv_ptrs(q, weight, bottom_diff != nullptr, false, "weight"));
    CHECK(check_conv_ptrs(q, bottom_diff, false, true, "bottom_diff"));
    CHECK(check_conv_ptrs(q, weight_diff, false, false, "weight_diff"));
    CHECK(check_conv_ptrs(q, bias_diff, false, false, "bias_diff"));
    CHECK(check_ws(workspace, ws_bytes, q.ws_both + pool_lrn_extra(q)));
    hipStream_t s = (hipStream_t)stream;
    char* ws = (char*)workspace;
    const float* relu_top = q.relu && !masked ? top : nullptr;
    if (!pool_lrn_staged(q)) {
        // the glue's backward into the workspace, then the layer's backward
        // on that gradient (already masked when relu_top was applied)
        float* gbuf = (float*)(ws + q.ws_both);
        LAUNCH(launch_lrn_pool_backward(pooled, lrn_top, lrn_top_diff, pool_mask, gbuf, q.N, q.K,
                                        q.Ho, q.Wo, PHo, PWo, pool->kernel_h, pool->kernel_w,
                                        pool->stride_h, pool->stride_w, pool->pad_h, pool->pad_w,
                                        lrn->local_size, lrn->alpha, lrn->beta, lrn->k, s,
                                        mask_u8),
               "fused LRN + pool backward launch");
        return caffe_conv_backward_ex(desc, gbuf, top, bottom, weight, bottom_diff, weight_diff,
                                      bias_diff, accumulate, flags, workspace, q.ws_both, stream,
                                      weight_stream);
    }
    hipStream_t wst = weight_stream != stream ? (hipStream_t)weight_stream : nullptr;
    if (q.N == 0) {
        if (bias_diff && !accumulate)
            LAUNCH(launch_fill_zero(bias_diff, q.K, s), "zero fill launch");
        if (weight_diff && !accumulate)
            LAUNCH(launch_fill_zero(weight_diff, q.weight_elems, s), "zero fill launch");
        return wst ? stream_follow(wst, s) : CAFFE_OK;
    }
    // the glue's backward written straight into the bf16 top-gradient
    // staging, with its bias-gradient partials
    float* sums = (float*)(ws + q.ws_both);
    LAUNCH(launch_lrn_pool_backward_bf16(pooled, lrn_top, lrn_top_diff, pool_mask, relu_top,
                                         (uint16_t*)(ws + q.off_dh), sums, q.N, q.K, q.Ho, q.Wo,
                                         PHo, PWo, pool->kernel_h, pool->kernel_w, pool->stride_h,
                                         pool->stride_w, pool->pad_h, pool->pad_w, lrn->local_size,
                                         lrn->alpha, lrn->beta, lrn->k, q.Kg, q.Kgp, q.G * q.Kgp,
                                         q.DHp, q.DWp, q.dtb, q.dlb, s, mask_u8),
           "fused LRN + pool backward staging launch");
    const int strips = lrn_pool_backward_strips(q.Ho, PHo, PWo, pool->kernel_h, pool->stride_h,
                                                pool->pad_h);
    return backward_bf16_staged(q, sums, q.N * strips, mask_bottom,
                                (flags & CAFFE_BACKWARD_BOTTOM_STAGED) != 0, bottom, weight,
                                bottom_diff, weight_diff, bias_diff, accumulate, ws, s, wst);
}

const char* caffe_status_string(int32_t status)
{
    switch (status) {
    case CAFFE_OK: return "CAFFE_OK";
    case CAFFE_ERR_INVALID_ARG: return "CAFFE_ERR_INVALID_ARG";
    case CAFFE_ERR_ALIGN: return "CAFFE_ERR_ALIGN";
    case CAFFE_ERR_WORKSPACE: return "CAFFE_ERR_WORKSPACE";
    case CAFFE_ERR_UNSUPPORTED: return "CAFFE_ERR_UNSUPPORTED";
    case CAFFE_ERR_HIP: return "CAFFE_ERR_HIP";
    default: return "CAFFE_ERR_UNKNOWN";
    }
}

const char* caffe_conv_status_string(int32_t status) { return caffe_status_string(status); }

size_t caffe_conv_workspace_bytes(const caffe_conv_desc* desc, int32_t pass)
{
    size_t bytes = 0;
    if (caffe_conv_workspace_size(desc, pass, &bytes) != CAFFE_OK)
        return SIZE_MAX;
    return bytes;
}

const char* caffe_last_error(void) { return g_err; }

int32_t caffe_version(void) { return 100; }

// ------------------------------------------------------------- glue layers
static int plan_pool(const caffe_pool_desc* d, int* Ho, int* Wo)
{
    if (!d)
        return fail(CAFFE_ERR_INVALID_ARG, "desc is NULL");
    if (d->N < 0 || d->C < 1 || d->H < 1 || d->W < 1 || d->kernel_h < 1 || d->kernel_w < 1 ||
        d->stride_h < 1 || d->stride_w < 1 || d->pad_h < 0 || d->pad_w < 0)
        return fail(CAFFE_ERR_INVALID_ARG, "bad pooling geometry");
    if (d->pad_h >= d->kernel_h || d->pad_w >= d->kernel_w)
        return fail(CAFFE_ERR_INVALID_ARG, "pad must be smaller than the kernel");
    if (d->H + 2 * (int64_t)d->pad_h < d->kernel_h || d->W + 2 * (int64_t)d->pad_w < d->kernel_w)
        return fail(CAFFE_ERR_INVALID_ARG, "kernel larger than the padded input");
    if (d->H > kMaxSpatial || d->W > kMaxSpatial || d->kernel_h > kMaxSpatial ||
        d->kernel_w > kMaxSpatial || d->stride_h > kMaxSpatial || d->stride_w > kMaxSpatial)
        return fail(CAFFE_ERR_UNSUPPORTED, "spatial sizes must be <= %d", kMaxSpatial);
    if ((int64_t)d->N * d->C * d->H * d->W * 4 > kMaxTensorBytes)
        return fail(CAFFE_ERR_UNSUPPORTED, "a tensor reaches 2^31 bytes");
    *Ho = (d->H + 2 * d->pad_h - d->kernel_h) / d->stride_h + 1;
    *Wo = (d->W + 2 * d->pad_w - d->kernel_w) / d->stride_w + 1;
    return CAFFE_OK;
}

int caffe_pool_out_shape(const caffe_pool_desc* desc, int32_t* Ho, int32_t* Wo)
{
    int ho, wo;
    CHECK(plan_pool(desc, &ho, &wo));
    if (!Ho || !Wo)
        return fail(CAFFE_ERR_INVALID_ARG, "Ho/Wo is NULL");
    *Ho = ho;
    *Wo = wo;
    return CAFFE_OK;
}

int caffe_maxpool_forward(const caffe_pool_desc* d, const float* bottom, float* top,
                          int32_t* mask, int32_t flags, void* stream)
{
    if (flags & ~CAFFE_POOL_RELU_INPUT)
        return fail(CAFFE_ERR_INVALID_ARG, "unknown pooling flags 0x%x", flags);
    int Ho, Wo;
    CHECK(plan_pool(d, &Ho, &Wo));
    const bool nz = d->N > 0;
    CHECK(check_ptr(bottom, nz, "bottom"));
    CHECK(check_ptr(top, nz, "top"));
    CHECK(check_ptr(mask, false, "mask"));
    LAUNCH(launch_maxpool_forward(bottom, top, mask, d->N * d->C, d->H, d->W, Ho, Wo, d->kernel_h,
                                  d->kernel_w, d->stride_h, d->stride_w, d->pad_h, d->pad_w,
                                  (flags & CAFFE_POOL_RELU_INPUT) ? 1 : 0, (hipStream_t)stream),
           "max-pool forward launch");
    return CAFFE_OK;
}

int caffe_maxpool_backward(const caffe_pool_desc* d, const float* top_diff, const int32_t* mask,
                           float* bottom_diff, void* stream)
{
    int Ho, Wo;
    CHECK(plan_pool(d, &Ho, &Wo));
    const bool nz = d->N > 0;
    CHECK(check_ptr(top_diff, nz, "top_diff"));
    CHECK(check_ptr(mask, nz, "mask"));
    CHECK(check_ptr(bottom_diff, nz, "bottom_diff"));
    LAUNCH(launch_maxpool_backward(top_diff, mask, bottom_diff, d->N * d->C, d->H, d->W, Ho, Wo,
                                   d->kernel_h, d->kernel_w, d->stride_h, d->stride_w, d->pad_h,
                                   d->pad_w, (hipStream_t)stream),
           "max-pool backward launch");
    return CAFFE_OK;
}

static int check_lrn(const caffe_lrn_desc* d)
{
    if (!d)
        return fail(CAFFE_ERR_INVALID_ARG, "desc is NULL");
    if (d->N < 0 || d->C < 1 || d->H < 1 || d->W < 1 || d->local_size < 1)
        return fail(CAFFE_ERR_INVALID_ARG, "bad LRN geometry");
    if (!(d->k > 0.f) || !(d->alpha >= 0.f) || !(d->beta >= 0.f))
        return fail(CAFFE_ERR_INVALID_ARG, "LRN needs k > 0, alpha >= 0, beta >= 0");
    if ((int64_t)d->N * d->C * d->H * d->W * 4 > kMaxTensorBytes)
        return fail(CAFFE_ERR_UNSUPPORTED, "a tensor reaches 2^31 bytes");
    return CAFFE_OK;
}

int caffe_lrn_forward(const caffe_lrn_desc* d, const float* bottom, float* top, void* stream)
{
    CHECK(check_lrn(d));
    const bool nz = d->N > 0;
    CHECK(check_ptr(bottom, nz, "bottom"));
    CHECK(check_ptr(top, nz, "top"));
    LAUNCH(launch_lrn_forward(bottom, top, d->N, d->C, d->H * d->W, d->local_size, d->alpha,
                              d->beta, d->k, (hipStream_t)stream),
           "LRN forward launch");
    return CAFFE_OK;
}

int caffe_lrn_backward(const caffe_lrn_desc* d, const float* bottom, const float* top,
                       const float* top_diff, float* bottom_diff, void* stream)
{
    CHECK(check_lrn(d));
    const bool nz = d->N > 0;
    CHECK(check_ptr(bottom, nz, "bottom"));
    CHECK(check_ptr(top, nz, "top"));
    CHECK(check_ptr(top_diff, nz, "top_diff"));
    CHECK(check_ptr(bottom_diff, nz, "bottom_diff"));
    LAUNCH(launch_lrn_backward(bottom, top, top_diff, bottom_diff, d->N, d->C, d->H * d->W,
                               d->local_size, d->alpha, d->beta, d->k, (hipStream_t)stream),
           "LRN backward launch");
    return CAFFE_OK;
}

static int check_pool_lrn(const caffe_pool_desc* pd, const caffe_lrn_desc* ld, int* Ho, int* Wo)
{
    CHECK(plan_pool(pd, Ho, Wo));
    CHECK(check_lrn(ld));
    if (ld->N != pd->N || ld->C != pd->C || ld->H != *Ho || ld->W != *Wo)
        return fail(CAFFE_ERR_INVALID_ARG, "the LRN blob (%d, %d, %d, %d) is not the pooled blob "
                    "(%d, %d, %d, %d)", ld->N, ld->C, ld->H, ld->W, pd->N, pd->C, *Ho, *Wo);
    if (!pool_lrn_fusable(pd->H, pd->W, *Ho, *Wo, pd->kernel_h, pd->stride_h, pd->pad_h,
                          ld->local_size))
        return fail(CAFFE_ERR_UNSUPPORTED, "fused pool + LRN needs local_size 3 or 5, W <= 256 "
                    "and at most 256 staged pooled positions");
    return CAFFE_OK;
}

int caffe_pool_lrn_forward(const caffe_pool_desc* pd, const caffe_lrn_desc* ld,
                           const float* bottom, float* pooled, int32_t* mask, float* top,
                           int32_t flags, void* stream)
{
    if (flags & ~(CAFFE_POOL_RELU_INPUT | CAFFE_POOL_MASK_OFFSETS))
        return fail(CAFFE_ERR_INVALID_ARG, "unknown pooling flags 0x%x", flags);
    int Ho, Wo;
    CHECK(check_pool_lrn(pd, ld, &Ho, &Wo));
    const int mask_u8 = (flags & CAFFE_POOL_MASK_OFFSETS) ? 1 : 0;
    if (mask_u8 && pd->kernel_h * pd->kernel_w > 255)
        return fail(CAFFE_ERR_UNSUPPORTED, "byte winner offsets need windows of at most 255 taps");
    const bool nz = pd->N > 0;
    CHECK(check_ptr(bottom, nz, "bottom"));
    CHECK(check_ptr(pooled, nz, "pooled"));
    CHECK(check_ptr(mask, false, "mask"));
    CHECK(check_ptr(top, nz, "top"));
    LAUNCH(launch_maxpool_forward(bottom, pooled, mask, pd->N * pd->C, pd->H, pd->W, Ho, Wo,
                                  pd->kernel_h, pd->kernel_w, pd->stride_h, pd->stride_w,
                                  pd->pad_h, pd->pad_w, (flags & CAFFE_POOL_RELU_INPUT) ? 1 : 0,
                                  (hipStream_t)stream, mask_u8),
           "max-pool forward launch");
    LAUNCH(launch_lrn_forward(pooled, top, ld->N, ld->C, ld->H * ld->W, ld->local_size, ld->alpha,
                              ld->beta, ld->k, (hipStream_t)stream),
           "LRN forward launch");
    return CAFFE_OK;
}

int caffe_pool_lrn_forward_into(const caffe_pool_desc* pd, const caffe_lrn_desc* ld,
                                const float* bottom, float* pooled, int32_t* mask, float* top,
                                int32_t flags, const caffe_conv_desc* next, void* next_workspace,
                                size_t next_ws_bytes, void* stream)
{
    if (flags & ~(CAFFE_POOL_RELU_INPUT | CAFFE_POOL_LRN_STAGE_ONLY | CAFFE_POOL_MASK_OFFSETS))
        return fail(CAFFE_ERR_INVALID_ARG, "unknown pooling flags 0x%x", flags);
    const bool write_top = !(flags & CAFFE_POOL_LRN_STAGE_ONLY);
    int Ho, Wo;
    CHECK(check_pool_lrn(pd, ld, &Ho, &Wo));
    const int mask_u8 = (flags & CAFFE_POOL_MASK_OFFSETS) ? 1 : 0;
    if (mask_u8 && pd->kernel_h * pd->kernel_w > 255)
        return fail(CAFFE_ERR_UNSUPPORTED, "byte winner offsets need windows of at most 255 taps");
    ConvPlan qn;
    if (!next)
        return fail(CAFFE_ERR_INVALID_ARG, "next is NULL");
    CHECK(plan_conv(next, &qn));
    if (qn.N != ld->N || qn.C != ld->C || qn.H != ld->H || qn.W != ld->W)
        return fail(CAFFE_ERR_INVALID_ARG, "the convolution's bottom (%d, %d, %d, %d) is not the "
                    "LRN's top (%d, %d, %d, %d)", qn.N, qn.C, qn.H, qn.W, ld->N, ld->C, ld->H,
                    ld->W);
    if (!caffe_hip_stage_from_lrn_ok(qn, ld->local_size))
        return fail(CAFFE_ERR_UNSUPPORTED, "the LRN's top cannot be staged for this convolution "
                    "(bf16 mode, channel groups of a multiple of 16 unpadded, LRN size 3 or 5)");
    CHECK(check_ws(next_workspace, next_ws_bytes, qn.ws_fwd));
    const bool nz = pd->N > 0;
    CHECK(check_ptr(bottom, nz, "bottom"));
    CHECK(check_ptr(pooled, nz, "pooled"));
    CHECK(check_ptr(mask, false, "mask"));
    CHECK(check_ptr(top, nz && write_top, "top"));
    hipStream_t s = (hipStream_t)stream;
    LAUNCH(launch_maxpool_forward(bottom, pooled, mask, pd->N * pd->C, pd->H, pd->W, Ho, Wo,
                                  pd->kernel_h, pd->kernel_w, pd->stride_h, pd->stride_w,
                                  pd->pad_h, pd->pad_w, (flags & CAFFE_POOL_RELU_INPUT) ? 1 : 0,
                                  s, mask_u8),
           "max-pool forward launch");
    uint16_t* xh = (uint16_t*)((char*)next_workspace + qn.off_xh_fwd);
    LAUNCH(launch_lrn_forward_stage(pooled, write_top ? top : nullptr, ld->N, ld->C, ld->H,
                                    ld->W, ld->local_size, ld->alpha, ld->beta, ld->k, xh, qn.XHp,
                                    qn.XWp, qn.ph, qn.pw, s),
           "LRN forward and staging launch");
    return CAFFE_OK;
}

int caffe_pool_lrn_stage_supported(const caffe_pool_desc* pd, const caffe_lrn_desc* ld,
                                   const caffe_conv_desc* next)
{
    int Ho, Wo;
    ConvPlan qn;
    if (check_pool_lrn(pd, ld, &Ho, &Wo) != CAFFE_OK || !next || plan_conv(next, &qn) != CAFFE_OK)
        return 0;
    return qn.N == ld->N && qn.C == ld->C && qn.H == ld->H && qn.W == ld->W &&
           caffe_hip_stage_from_lrn_ok(qn, ld->local_size);
}

int caffe_lrn_pool_backward(const caffe_pool_desc* pd, const caffe_lrn_desc* ld,
                            const float* pooled, const float* top, const float* top_diff,
                            const int32_t* mask, float* bottom_diff, void* stream)
{
    return caffe_lrn_pool_backward_ex(pd, ld, pooled, top, top_diff, mask, bottom_diff, 0, stream);
}

int caffe_lrn_pool_backward_ex(const caffe_pool_desc* pd, const caffe_lrn_desc* ld,
                               const float* pooled, const float* top, const float* top_diff,
                               const int32_t* mask, float* bottom_diff, int32_t flags,
                               void* stream)
{
    if (flags & ~CAFFE_BACKWARD_POOL_MASK_OFFSETS)
        return fail(CAFFE_ERR_INVALID_ARG, "unknown flags 0x%x", flags);
    const int mask_u8 = flags ? 1 : 0;
    int Ho, Wo;
    CHECK(check_pool_lrn(pd, ld, &Ho, &Wo));
    if (mask_u8 && pd->kernel_h * pd->kernel_w > 255)
        return fail(CAFFE_ERR_UNSUPPORTED, "byte winner offsets need windows of at most 255 taps");
    const bool nz = pd->N > 0;
    CHECK(check_ptr(pooled, nz, "pooled"));
    CHECK(check_ptr(top, nz, "top"));
    CHECK(check_ptr(top_diff, nz, "top_diff"));
    CHECK(check_ptr(mask, nz, "mask"));
    CHECK(check_ptr(bottom_diff, nz, "bottom_diff"));
    LAUNCH(launch_lrn_pool_backward(pooled, top, top_diff, mask, bottom_diff, pd->N, pd->C, pd->H,
                                    pd->W, Ho, Wo, pd->kernel_h, pd->kernel_w, pd->stride_h,
                                    pd->stride_w, pd->pad_h, pd->pad_w, ld->local_size, ld->alpha,
                                    ld->beta, ld->k, (hipStream_t)stream, mask_u8),
           "fused LRN + pool backward launch");
    return CAFFE_OK;
}

int caffe_relu_backward(const float* top, const float* top_diff, float* bottom_diff,
                        int64_t count, void* stream)
{
    if (count < 0)
        return fail(CAFFE_ERR_INVALID_ARG, "count must be >= 0");
    if (count * 4 > kMaxTensorBytes)
        return fail(CAFFE_ERR_UNSUPPORTED, "a tensor reaches 2^31 bytes");
    const bool nz = count > 0;
    CHECK(check_ptr(top, nz, "top"));
    CHECK(check_ptr(top_diff, nz, "top_diff"));
    CHECK(check_ptr(bottom_diff, nz, "bottom_diff"));
    LAUNCH(launch_relu_mask(top_diff, top, bottom_diff, count, (hipStream_t)stream),
           "ReLU backward launch");
    return CAFFE_OK;
}

int caffe_cast_f32_to_bf16(const float* in, uint16_t* out, int64_t count, void* stream)
{
    if (count < 0)
        return fail(CAFFE_ERR_INVALID_ARG, "count < 0");
    CHECK(check_ptr(in, count > 0, "in"));
    CHECK(check_ptr(out, count > 0, "out"));
    LAUNCH(launch_cast_f32_bf16(in, out, count, (hipStream_t)stream), "cast launch");
    return CAFFE_OK;
}

// ------------------------------------------------------------- solver
int caffe_sgd_learning_rate(const caffe_lr_schedule* sc, int64_t iter, float* lr)
{
    if (!sc || !lr)
        return fail(CAFFE_ERR_INVALID_ARG, "schedule or lr is NULL");
    if (iter < 0)
        return fail(CAFFE_ERR_INVALID_ARG, "iteration %lld < 0", (long long)iter);
    if (!(sc->base_lr >= 0.f))
        return fail(CAFFE_ERR_INVALID_ARG, "base_lr must be >= 0");
    const double base = sc->base_lr, gamma = sc->gamma, t = (double)iter;
    double r;
    switch (sc->policy) {
    case CAFFE_LR_FIXED:
        r = base;
        break;
    case CAFFE_LR_STEP:
        if (sc->stepsize < 1)
            return fail(CAFFE_ERR_INVALID_ARG, "step schedule needs stepsize >= 1");
        r = base * std::pow(gamma, (double)(iter / sc->stepsize));
        break;
    case CAFFE_LR_EXP:
        r = base * std::pow(gamma, t);
        break;
    case CAFFE_LR_INV:
        r = base * std::pow(1.0 + gamma * t, -(double)sc->power);
        break;
    default:
        return fail(CAFFE_ERR_INVALID_ARG, "unknown learning-rate policy %d", sc->policy);
    }
    if (!std::isfinite(r) || !std::isfinite((float)r))
        return fail(CAFFE_ERR_INVALID_ARG, "learning rate is not finite at iteration %lld",
                    (long long)iter);
    *lr = (float)r;
    return CAFFE_OK;
}

int caffe_softmax_loss(const float* scores, const int32_t* labels, int32_t N, int32_t K,
                       float loss_weight, float* loss, float* sample_loss, float* prob,
                       float* scores_diff, void* stream)
{
    if (N < 0 || K < 1 || K > (1 << 24))
        return fail(CAFFE_ERR_INVALID_ARG, "softmax loss needs N >= 0 and 1 <= K <= 2^24");
    if ((int64_t)N * K * 4 > kMaxTensorBytes)
        return fail(CAFFE_ERR_UNSUPPORTED, "a tensor reaches 2^31 bytes");
    if (!std::isfinite(loss_weight))
        return fail(CAFFE_ERR_INVALID_ARG, "loss_weight is not finite");
    const bool nz = N > 0;
    CHECK(check_ptr(scores, nz, "scores"));
    CHECK(check_ptr(labels, nz, "labels"));
    CHECK(check_ptr(loss, true, "loss"));
    CHECK(check_ptr(sample_loss, nz, "sample_loss"));
    CHECK(check_ptr(prob, false, "prob"));
    CHECK(check_ptr(scores_diff, false, "scores_diff"));
    LAUNCH(launch_softmax_loss(scores, labels, N, K, loss_weight, loss, sample_loss, prob,
                               scores_diff, (hipStream_t)stream),
           "softmax loss launch");
    return CAFFE_OK;
}

int caffe_sgd_update(float* w, const float* g, float* v, int64_t count, float lr, float momentum,
                     float weight_decay, void* stream)
{
    if (count < 0)
        return fail(CAFFE_ERR_INVALID_ARG, "count < 0");
    if (!std::isfinite(lr) || !std::isfinite(momentum) || !std::isfinite(weight_decay))
        return fail(CAFFE_ERR_INVALID_ARG, "lr, momentum and weight_decay must be finite");
    const bool nz = count > 0;
    CHECK(check_ptr(w, nz, "w"));
    CHECK(check_ptr(g, nz, "g"));
    CHECK(check_ptr(v, nz, "v"));
    LAUNCH(launch_sgd_update(w, g, v, count, lr, nullptr, momentum, weight_decay,
                             (hipStream_t)stream),
           "SGD update launch");
    return CAFFE_OK;
}

int caffe_sgd_update_device_lr(float* w, const float* g, float* v, int64_t count, const float* lr,
                               float momentum, float weight_decay, void* stream)
{
    if (count < 0)
        return fail(CAFFE_ERR_INVALID_ARG, "count < 0");
    if (!std::isfinite(momentum) || !std::isfinite(weight_decay))
        return fail(CAFFE_ERR_INVALID_ARG, "momentum and weight_decay must be finite");
    const bool nz = count > 0;
    CHECK(check_ptr(w, nz, "w"));
    CHECK(check_ptr(g, nz, "g"));
    CHECK(check_ptr(v, nz, "v"));
    if (nz && !lr)
        return fail(CAFFE_ERR_INVALID_ARG, "lr is NULL");
    if (lr && !aligned(lr, 4))
        return fail(CAFFE_ERR_ALIGN, "lr is not 4-byte aligned");
    LAUNCH(launch_sgd_update(w, g, v, count, 0.f, lr, momentum, weight_decay, (hipStream_t)stream),
           "SGD update launch");
    return CAFFE_OK;
}

}  // extern "C"
