// kernels.h -- host-side view of the gfx950 kernels: parameter blocks and
// launchers.  Shapes are validated by the C ABI layer (api.cpp) before any
// launcher runs; launchers trust their arguments.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace caffe_hip {

// Unsigned division by a runtime constant d >= 1 for numerators < 2^31:
// q = (x * mul) >> shift with shift = 31 + ceil(log2 d), mul = ceil(2^shift / d).
struct FastDiv {
    uint32_t d, mul, shift;
};
FastDiv make_fastdiv(uint32_t d);

// Bytes of the library's static per-device scratch array (the workspace of
// caffe_conv_forward_noalloc) and the current device's address of it, looked
// up on the first call on each device.
constexpr size_t kStaticScratchBytes = size_t(64) << 20;
hipError_t static_scratch_address(void** ptr);

// Implicit GEMM whose reduction index r = (c, u, v) walks a kh x kw window of
// a gather source X[N][Cin][IH][IW] and whose column index walks the output
// grid (n, i, j) in N x OH x OW:
//   C_g[m][col] = sum_r A[g][r][m] * X[n][g*Cin_g + c][i*sh - ph + u][j*sw - pw + v]
// A is laid out [G][R][M] (m contiguous): both operands are copied from
// global memory straight into LDS, 64 consecutive elements of one k row per
// wave copy.
// epi == 0 (forward): Y[n][g*M + m][i][j] = [relu](C + bias[g*M + m])
// epi == 1 (data gradient, phase-stacked): row m = (c, fh, fw) and
//   Y[n][g*Cg_out + c][psh*(i + a0h) + fh - oph][psw*(j + a0w) + fw - opw] = C
//   for in-range positions (each output element is written exactly once).
// Omask (epi 1 only, may be null): a float tensor laid out like Y; each
// result is stored as 0 wherever Omask is not > 0 (the backward of a ReLU
// whose output the gradient flows into).
struct ConvGemmParams {
    const void* A;
    const void* X;
    const float* Omask;
    float* Y;
    const float* bias;
    uint32_t A_bytes, X_bytes, Y_bytes;
    int N, Cin, IH, IW, Cin_g;
    int kh, kw, sh, sw, ph, pw;
    int OH, OW;
    int M, R, G;
    int Ncol;
    int relu;
    int Cout, OutH, OutW;
    int psh, psw, a0h, a0w, oph, opw, Cg_out;
    int blocked;    // channel-blocked reduction order (else tap-major), with tap_major
    int xcd_order;  // XCD-contiguous tile order (else linear)
    // 1: unit order instead (every row and column tile of one (group, split)
    // unit on one XCD, units dealt round-robin over the XCDs; the grid is
    // whole rounds of 8 units, see wgrad_grid)
    int unit_order;
    int splits, stages_per_split;  // dense split-K GEMM only
    FastDiv div_pss, div_psw;  // epi 1: phases psh*psw and psw
    // epi 0 / 1, tail_splits > 1: the tiles from tail_T on (whole column
    // tiles of the last group, its columns from tail_c0 on) run as
    // tail_splits reduction ranges of tail_sps stages, each storing its
    // partial Pt[split][m][col - tail_c0] (Ncol - tail_c0 columns) for
    // launch_conv_split_reduce_* over that region to finish
    int tail_T, tail_splits, tail_sps, tail_c0;
    float* Pt;
    uint32_t Pt_bytes;
    // channel-major gathered operand (r = (c, u, v)) only, optional: byte
    // offsets (c*IH*IW + u*IW + v) * 4 of the taps r < R, then X_bytes up to
    // a whole number of stages (see launch_tap_table)
    const uint32_t* taps;
};

// Dense split-K GEMM on the same core (the inner-product layer):
//   P[s][m][col] = sum_{r in split s} A[r][m] * X[r][col]
// A is [R][M] and X is [R][Ncol] (row-major, G = 1); split s covers the
// reduction stages s*stages_per_split .. (s+1)*stages_per_split - 1; Y is P.
hipError_t launch_dense_gemm_f32(const ConvGemmParams& p, int tile, hipStream_t s);
// Dense split-K GEMM with reduction-contiguous operands: P[split][m][n] =
// sum_r A[m][r] B[n][r] (A = p.A [M][R], B = p.X [Ncol][R], P = p.Y).
// R % 4 == 0 and 16-byte aligned A and B, else hipErrorInvalidValue.
hipError_t launch_dense_gemm_nt_f32(const ConvGemmParams& p, int tile, hipStream_t s);
// Compute units of the current device; 256 when no device answers.
int device_cu_count();

// out[c][r] = in[r][c] for an R x C row-major float matrix.
hipError_t launch_transpose_f32(const float* in, float* out, int R, int C, hipStream_t s);

// D = G [Y > 0] element by element.
hipError_t launch_relu_mask(const float* G, const float* Y, float* D, int64_t count, hipStream_t s);
// out[i] = act(sum_{s < splits} P[s*count + i] + bias[i % ncol]) in a fixed
// order (bias may be null; act = ReLU when relu), stored as 0 where a non-null
// mask is not > 0.
hipError_t launch_split_reduce(const float* P, int splits, int count, int ncol, const float* bias,
                               int relu, const float* mask, float* out, hipStream_t s);
// The epilogues of split convolution GEMMs, from the partials
// P[split][g][m][col] (col = n * OHW + pix of the GEMM's output grid), each
// output's partials added in split order:
//   forward: Y[n][g*M + m][pix] = act(bias[g*M + m] + sum_s P[s][g][m][col])
//   data gradient (phase-stacked rows m = (c, fh, fw)): dX[n][g*Cg_out + c]
//   [psh (a + a0h) - oph + fh][psw (b + a0w) - opw + fw] = sum_s P[s][g][m][col]
//   (pix = a * OW + b; positions outside the image are dropped), times
//   [mask > 0] where mask is non-null.
// With g0 / c0, only the outputs of groups g0.. and columns c0.. (the region
// a tail split covers), from P[split][g - g0][m][col - c0].
hipError_t launch_conv_split_reduce_fwd(const float* P, int splits, const ConvGemmParams& q,
                                        float* Y, hipStream_t s, int g0 = 0, int c0 = 0);
hipError_t launch_conv_split_reduce_dgrad(const float* P, int splits, const ConvGemmParams& q,
                                          const float* mask, float* dX, hipStream_t s,
                                          int g0 = 0, int c0 = 0);

// Split-K weight gradient:
//   P[s][g*Kg + m][r] = sum_{col in split s} D[n][g*Kg + m][i][j] * X[n][g*Cg + c][i*sh - ph + u][j*sw - pw + v]
// When dbp is given, the workgroups of the first tap tile also write
// dbp[s][g*Kg + m] = sum_{col in split s} D (the bias-gradient partials).
struct WgradParams {
    const void* D;
    const void* X;
    float* P;
    float* dbp;
    uint32_t D_bytes, X_bytes, P_bytes;
    int N, C, IH, IW, Cg, K, Kg;
    int kh, kw, sh, sw, ph, pw;
    int OH, OW;
    int R, G;
    int Ncol, cols_per_split, splits;
    FastDiv div_ohw, div_ow;
    int xcd_order;  // XCD-contiguous tile order (else linear)
    // 1: unit order instead (every row and column tile of one (group, split)
    // unit on one XCD, units dealt round-robin over the XCDs; the grid is
    // whole rounds of 8 units, see wgrad_grid)
    int unit_order;
    // quad-order kernel only: the per-column table (see
    // launch_wgrad_col_table) and the element shift of X's resource base
    const void* T;
    uint32_t T_bytes;
    int xpad;
};

// Tile shapes a launcher may pick; see conv_gemm.hip.
enum GemmTile : int {
    TILE_128x128 = 0,      // 32x32x2 MFMA, 4 waves as 2x2, each 64x64, 16-deep stages
    TILE_96x256 = 1,       // 32x32x2 MFMA, 4 waves as 1x4, each 96x64
    TILE_48x256 = 2,       // 16x16x4 MFMA, 4 waves as 1x4, each 48x64
    TILE_64x256 = 3,       // 32x32x2 MFMA, 4 waves as 1x4, each 64x64
    TILE_128x128_K32 = 4,  // as TILE_128x128 with 32-deep stages
    TILE_COUNT
};
int gemm_tile_m(int tile);
int gemm_tile_n(int tile);
int gemm_tile_k(int tile);  // reduction depth of one pipeline stage

// Smallest stage depth of any tile: channel counts divisible by it can use
// the tap-major order with some tile.
constexpr int kGemmMinTK = 16;

// tap_major: the reduction index runs in the channel-blocked order
// r = (c / TK, u, v, c % TK), TK = gemm_tile_k(tile), or tap-major
// r = (u, v, c) (A packed to match, see launch_pack_weights); needs
// Cin_g % TK == 0.  Otherwise r = (c, u, v).
// epi 0: forward epilogue (bias, ReLU, NCHW store); epi 1: data-gradient
// scatter (with p.Omask, the bottom mask); epi 3: the same gathered GEMM cut
// into p.splits reduction ranges of p.stages_per_split stages, each storing
// its partial P[split][g][m][col] to p.Y (see launch_conv_split_reduce_*).
hipError_t launch_conv_gemm_f32(const ConvGemmParams& p, int epi, int tile, bool tap_major,
                                hipStream_t s);

// Tap offsets of the channel-major order r = c*kh*kw + u*kw + v:
// T[r] = (c*IHW + u*IW + v) * 4 for r < R, T[r] = oob for R <= r < rpad.
hipError_t launch_tap_table(uint32_t* T, int rpad, int R, int kh, int kw, int IHW, int IW,
                            uint32_t oob, hipStream_t s);

// Forward weights W[G*M][Cg][khw] -> Wp[g][r][m] in the reduction order
// r = ((c / tk) * khw + t) * tk + c % tk (order > 0), r = t * Cg + c
// (order < 0) or r = c * khw + t (order == 0), t = u*kw + v.
hipError_t launch_pack_weights(const float* W, float* Wp, int G, int M, int Cg, int khw, int tk,
                               int order, hipStream_t s);

enum WgradTile : int {
    WTILE_128x128 = 0,  // 4 waves as 2x2, each 64x64
    WTILE_96x128 = 1,   // 4 waves as 1x4, each 96x32
    WTILE_64x128 = 2,   // 4 waves as 2x2, each 32x64
    WTILE_COUNT
};
int wgrad_tile_m(int tile);
int wgrad_tile_n(int tile);
int wgrad_tile_k();
hipError_t launch_conv_wgrad_f32(const WgradParams& p, int tile, hipStream_t s);

// Quad-order weight gradient (see conv_wgrad.hip): Cg % 4 == 0 and a 3x3 or
// 5x5 kernel; reads p.T, written by launch_wgrad_col_table for the same
// geometry.  Partials in the layout launch_conv_wgrad_f32 writes.
bool wgrad_quad_supported(int Cg, int kh, int kw);
hipError_t launch_conv_wgrad_quad_f32(const WgradParams& p, int tile, hipStream_t s);
// The same GEMM with both operands copied global -> LDS by LDS DMA (same
// table, same conditions, cols_per_split a multiple of 16).
hipError_t launch_conv_wgrad_dma_f32(const WgradParams& p, int tile, hipStream_t s);
// Three words per output column col < ncol_pad (ncol_pad a multiple of 16):
// {byte offset of the column's window origin in X plus xpad = ph*IW + pw
// elements, mask of the window's taps u*kw + v that lie outside the image,
// byte offset of the column in D's channel 0}; columns past ncol get
// {2^31, ~0, 2^31}.
hipError_t launch_wgrad_col_table(uint32_t* T, int ncol, int ncol_pad, int C, int IH, int IW,
                                  int K, int OH, int OW, int kh, int kw, int sh, int sw, int ph,
                                  int pw, hipStream_t s);

// ---- bf16 operands (conv_bf16.hip) ----
// Reduction depth of a bf16 implicit-GEMM stage (8 chunks of 8 bf16: 128
// bytes of each operand row); the packed reductions Rp and Rtp are padded to
// multiples of it.
constexpr int kBf16TK = 64;

// bf16 implicit-GEMM tiles (rows x columns per workgroup).  The 8-wave
// shapes run two waves per SIMD on the LDS-bound GEMM: measured 2-12% faster
// than the same tile with 4 waves (CaffeNet conv1-5 at N=512).
enum Bf16Tile {
    BTILE_128x256 = 0,  // 32x32x16 MFMA, 8 waves as 2 x 4, each 64x64
    BTILE_96x256 = 1,   // 32x32x16, 8 waves as 1 x 8, each 96x32
    BTILE_64x256 = 2,   // 32x32x16, 4 waves as 1 x 4, each 64x64
    BTILE_48x256 = 3,   // 16x16x32 MFMA, 8 waves as 1 x 8, each 48x32
    BTILE_COUNT
};
int bf16_tile_m(int tile);
// Pipeline of the bf16 implicit GEMM (kBf16TK-deep stages): LDS buffers.
enum Bf16Pipe {
    BPIPE_2 = 0,  // double-buffered
    BPIPE_3 = 1,  // three buffers (copies two stages ahead)
    BPIPE_COUNT
};

// Implicit GEMM over a channel-contiguous, zero-bordered bf16 gather source
// X[N][IHp][IWp][Ctot] whose group g owns channels g*Cgp .. g*Cgp + Cgp - 1.
// The reduction r = (u, v, c) over kh x kwp x Cgp runs in 16-byte chunks of 8
// consecutive elements, KC = kh * kwg * Cg8 of them:
//  - Cgp a multiple of 8: a chunk is 8 channels of one tap; Cg8 = Cgp / 8
//    chunks per tap, kwg = kw taps per kernel row, vstr = Ctot;
//  - Cgp in {1, 2, 4} (one group, Ctot = Cgp): a chunk is 8 / Cgp
//    horizontally adjacent taps of all Cgp channels (the staged row is
//    contiguous along (v, c)); Cg8 = 1, kwg = kwp / (8 / Cgp) tap groups per
//    kernel row, vstr = 8.
// Chunk kc = (u, vg, c8) (c8 fastest) lies (u*IWp*Ctot + vg*vstr + 8*c8)
// elements from its column's pixel.  A is [G*M][Rp] bf16 (Rp >= 8*KC a
// multiple of kBf16TK, zero past 8*KC and at taps past kw).
//   C_g[m][col] = sum_r A[g*M + m][r] * X[n][i*sh + oh0 + u][j*sw + ow0 + v][g*Cgp + c]
// for col = (n, i, j) in N x OH x OW: the borders of X stand for the
// convolution's zero padding, so every gathered position lies inside it.
// Epilogues as ConvGemmParams (epi 0 forward, epi 1 phase-stacked data
// gradient); Omask (epi 1, may be null) is a tensor laid out like Y of bf16
// values, or of floats (omask_f32) that count as the bf16 they round to.
struct GemmBf16Params {
    const uint16_t* A;
    const uint16_t* X;
    const void* Omask;
    int omask_f32;
    float* Y;
    const float* bias;
    uint32_t A_bytes, X_bytes, Y_bytes;
    int N, IHp, IWp, Ctot, Cgp, Cg8, KC, vstr;
    int kh, kw, sh, sw, oh0, ow0;  // kw: tap groups per kernel row (kwg)
    int OH, OW;
    int M, Rp, G, Ncol;
    int relu;
    int Cout, OutH, OutW;
    int psh, psw, a0h, a0w, oph, opw, Cg_out;
    int xcd_order;
    FastDiv div_cg8, div_kw;
    // blocked: the reduction runs over 64-channel blocks outer, taps inner
    // (stage t = block t / ntap of tap t % ntap; A packed in that order), so
    // that the workgroups of one XCD share fewer staged rows at a time
    // (needs Cgp % 64 == 0 and one tap per tap group)
    int blocked, ntap;
    FastDiv div_ntap;
    // epilogue divisions: output pixels per image and per row (epi 0 and 1),
    // phases psh*psw and psw (epi 1)
    FastDiv div_ohw, div_ow, div_pss, div_psw;
    // epi 2 (a stride-1 data gradient whose output grid is the image, taken
    // as the top gradient of the layer below): instead of Y, each value v of
    // channel c = g*Cg_out + m at pixel (n, h, w), masked as in epi 1, goes
    // to Sh[n][h + s_tb][w + s_lb][c] as bf16 (nearest even) -- the layer
    // below's staged top gradient, s_Ktot channels -- and each wave's sum of
    // its 64 columns' float values to Ssum[c * s_T + 4 * column tile + wave
    // column] (the bias gradient's partial sums, s_T per channel)
    uint16_t* Sh;
    float* Ssum;
    uint32_t Sh_bytes, Ssum_bytes;
    int s_Hp, s_Wp, s_tb, s_lb, s_Ktot, s_T;
};
hipError_t launch_conv_gemm_bf16(const GemmBf16Params& p, int epi, int tile, int pipe,
                                 hipStream_t s);
// Terms per channel of the epi 2 bias partial sums for an image grid of
// ncol pixels (4 per 256-column tile).
int stage_below_terms(int64_t ncol);
// Zero the border (every pixel outside rows tb .. tb + H - 1 and columns
// lb .. lb + W - 1) of an N x DHp x DWp x Ktot bf16 staging.
hipError_t launch_dh_zero_border(uint16_t* Dh, int N, int DHp, int DWp, int tb, int lb, int H,
                                 int W, int Ktot, hipStream_t s);

// Split-K weight gradient over channel-contiguous, zero-bordered bf16
// operands (D laid out [N][DHp][DWp][Ktot] with the real pixels at offset
// (dtb, dlb); X as in GemmBf16Params with oh0 = ow0 = 0):
//   P[s][g*Kg + m][(u*kwp + v)*Cgp + c] =
//       sum_{col in split s} D[n][i + dtb][j + dlb][g*Kgp + m] * X[n][i*sh + u][j*sw + v][g*Cgp + c]
// with col = (n, i, j) and Rw = kh*kwp*Cgp columns per output channel (kw
// below holds kwp: kw rounded up to the taps of a chunk).
struct WgradBf16Params {
    const uint16_t* D;
    const uint16_t* X;
    float* P;
    uint32_t D_bytes, X_bytes, P_bytes;
    int N, IHp, IWp, Ctot, Cgp, K, Kg, Kgp, Ktot;
    int DHp, DWp, dtb, dlb;
    int kh, kw, sh, sw;
    int OH, OW;
    int Rw, G;
    int Ncol, cols_per_split, splits;
    FastDiv div_ohw, div_ow;
    // 1: the blocks of one (group, split) unit -- every row and column tile,
    // all reading the same top-gradient and input slab -- run on one XCD,
    // units dealt round-robin over the 8 XCDs, so that the slab is fetched
    // from HBM once into that XCD's L2
    int unit_order;
};
constexpr int kBf16WgradTK = 64;  // output pixels per weight-gradient stage
// bf16 weight-gradient tiles (output channels x reduction indices r); with
// 8 waves rather than 4, measured equal or up to 5% faster per layer
enum Bf16WgradTile {
    BWTILE_128x256 = 0,  // 8 waves as 2x4, each 64x64
    BWTILE_96x256 = 1,   // 8 waves as 1x8, each 96x32
    BWTILE_COUNT
};
int bf16_wgrad_tile_m(int tile);
constexpr int kBf16WgradTN = 256;
// cols_per_split must be a multiple of kBf16WgradTK
hipError_t launch_conv_wgrad_bf16(const WgradBf16Params& p, int tile, hipStream_t s);

// dW[k][c][u][v] = (accumulate ? dW : 0) + sum_s P[s][k][(bu*kwp + bv)*Cgp + cp]
// for c < Cg, u < kh, v < kw (fixed order), (bu, bv, cp) from (u, v, c) as in
// launch_pack_weights_bf16.
hipError_t launch_wgrad_reduce_perm(const float* P, float* dW, int K, int Rw, int Cgp, int Cg,
                                    int kh, int kw, int kwp, int S, int splits, int accumulate,
                                    hipStream_t s);

// Xp[n][hp][wp][g*Cgp + c] = X[n][g*Cg + c][hp - tb][wp - lb] inside the H x W
// image (c < Cg), else 0: the zero-bordered channel-contiguous copy, Hp x Wp
// pixels per image; Ctot = G*Cgp, a multiple of 8, or Cgp in {1, 2, 4} with
// G = 1 and Hp*Wp a multiple of 8 / Cgp.  X holds bf16 values, or floats
// (x_f32) that are rounded to bf16 (nearest-even) on the way.
hipError_t launch_stage_nhwc_bf16(const void* X, int x_f32, uint16_t* Xp, int N, int C, int H,
                                  int W, int Cg, int Cgp, int Ctot, int Hp, int Wp, int tb, int lb,
                                  hipStream_t s);

// Dh[n][hp][wp][g*Kgp + k] = bf16(relu ? G [Y > 0] : G)[n][g*Kg + k][hp - tb][wp - lb]
// inside the H x W grid (k < Kg), else 0.  sums (may be null): the fp32
// bias-gradient partials, sums[k*T + t] for T = diff_prep_terms(N, Hp*Wp)
// terms per output channel (one per run of 512 bordered pixels of an image,
// t = image * runs + run).
int diff_prep_terms(int N, int HWp);
hipError_t launch_diff_prep_bf16(const float* G, const float* Y, uint16_t* Dh, float* sums, int N,
                                 int K, int H, int W, int Kg, int Kgp, int Ktot, int Hp, int Wp,
                                 int tb, int lb, int relu, hipStream_t s);

// db[k] = (accumulate ? db[k] : 0) + sum_{t < T} sums[k*T + t] (fixed order).
hipError_t launch_bias_reduce(const float* sums, float* db, int T, int K, int accumulate,
                              hipStream_t s);

// Wp[o][(bu*kwp + bv)*Cgp + cp] = W[o][c][u][v], 0 outside the kernel and the
// channels and past the staged taps; plain staging (S = 1): (bu, bv, cp) =
// (u, v, c); space-to-depth by S: u = S*bu + fu, v = S*bv + fv,
// cp = (fu*S + fv)*Cg + c.
hipError_t launch_pack_weights_bf16(const uint16_t* W, uint16_t* Wp, int K, int Cg, int Cgp,
                                    int kh, int kw, int kwp, int S, int Rp, hipStream_t s);
// Space-to-depth staging by S of one group of C channels:
// Xp[n][a][b][(fu*S + fv)*C + c] = X[n][c][S*a + fu - ph][S*b + fv - pw] (0
// outside the image and for staged channels past C*S*S, up to Csp, a
// multiple of 8), XHp x XWp staged pixels per image.  X holds bf16 values, or
// floats (x_f32) rounded to bf16 on the way.
hipError_t launch_stage_s2d_bf16(const void* X, int x_f32, uint16_t* Xp, int N, int C, int H,
                                 int W, int S, int ph, int pw, int XHp, int XWp, int Csp,
                                 hipStream_t s);

// Wt[g][(c, fh, fw)][(th*Tw + tw)*Kgp + k] = W[g*Kg + k][c][fh + sh*(Th-1-th)][fw + sw*(Tw-1-tw)]
// (0 past the kernel edge, for k >= Kg and past Th*Tw*Kgp); blocked (Kgp % 64
// == 0): the index ((k / 64)*Th*Tw + th*Tw + tw)*64 + k % 64 instead.
hipError_t launch_dgrad_weights_bf16(const uint16_t* W, uint16_t* Wt, int G, int Kg, int Kgp,
                                     int Cg, int kh, int kw, int sh, int sw, int Th, int Tw,
                                     int Rtp, int blocked, hipStream_t s);

// D = relu ? G * [Y > 0] : G (written to D unless D is null) and, unless
// plane_sums is null, plane_sums[p] = sum of D over plane p (fixed order).
hipError_t launch_relu_mask_bias(const float* G, const float* Y, float* D, float* plane_sums,
                                 int planes, int plane_size, int relu, hipStream_t s);

// Wt[g][r][(c, fh, fw)] = W[g*Kg + k][c][fh + sh*(Th-1-th)][fw + sw*(Tw-1-tw)]
// (0 where the tap index passes the kernel edge; m = (c, fh, fw) contiguous),
// r = (k, th, tw), the channel-blocked r = (k / tk, th, tw, k % tk) when
// tk > 0, or the tap-major r = (th, tw, k) when tk < 0.
hipError_t launch_dgrad_weight_transform(const float* W, float* Wt, int G, int Kg, int Cg, int kh,
                                         int kw, int sh, int sw, int Th, int Tw, int tk,
                                         hipStream_t s);

// out[i] = (accumulate ? out[i] : 0) + sum_{s < splits} P[s*count + i]   (fixed order)
// and, if db != null, db[k] = (accumulate ? db[k] : 0) + sum_{n < N} plane_sums[n*K + k].
hipError_t launch_wgrad_reduce(const float* P, float* out, int count, int splits,
                               const float* plane_sums, float* db, int N, int K, int accumulate,
                               hipStream_t s);

hipError_t launch_fill_zero(float* out, int64_t count, hipStream_t s);

// Glue layers (layers.hip).
// relu_input: windows whose maximum is not > 0 record mask -1 (no winner),
// so the backward pass routes them nothing.
// (mask_u8: mask is bytes, each winner's offset du * kw + dv in its window,
// 255 for none)
hipError_t launch_maxpool_forward(const float* x, float* y, int32_t* mask, int NC, int H, int W,
                                  int OH, int OW, int kh, int kw, int sh, int sw, int ph, int pw,
                                  int relu_input, hipStream_t s,
                                  int mask_u8 = 0);
hipError_t launch_maxpool_backward(const float* dy, const int32_t* mask, float* dx, int NC, int H,
                                   int W, int OH, int OW, int kh, int kw, int sh, int sw, int ph,
                                   int pw, hipStream_t s);
// launch_lrn_forward whose output also goes, rounded to bf16, to the
// zero-bordered staging Xp[n][h + tb][w + lb][c] (Hp x Wp pixels of C
// channels, border written too) of a convolution that takes it as its
// bottom; C a multiple of 16, size 3 or 5.
hipError_t launch_lrn_forward_stage(const float* x, float* y, int N, int C, int H, int W,
                                    int size, float alpha, float beta, float k, uint16_t* Xp,
                                    int Hp, int Wp, int tb, int lb, hipStream_t s);
hipError_t launch_lrn_forward(const float* x, float* y, int N, int C, int HW, int size,
                              float alpha, float beta, float k, hipStream_t s);
hipError_t launch_lrn_backward(const float* x, const float* y, const float* dy, float* dx, int N,
                               int C, int HW, int size, float alpha, float beta, float k,
                               hipStream_t s);
// The backward of max-pool then LRN in one pass (no pooled gradient in HBM).
// LRN sizes 3 and 5; the geometry must pass pool_lrn_fusable
// (hipErrorInvalidValue otherwise).
bool pool_lrn_fusable(int H, int W, int OH, int OW, int kh, int sh, int ph, int size);
// Row strips of the fused LRN + max-pool backward (0: not fusable).
int lrn_pool_backward_strips(int H, int OH, int OW, int kh, int sh, int ph);
// (Both fused backward launchers take the LRN's output `top` for the
// interface only: the kernels form it again from `pooled`, bit for bit.
// mask_u8: the mask as launch_maxpool_forward writes it with mask_u8.)
// The fused backward written as the bf16 top-gradient staging of the
// convolution below (channels in groups of Kg, each padded to Kgp, Ktot in
// all, on a DHp x DWp grid with the image at (tb, lb)), plus the grid's zero
// border and the bias-gradient partials sums[c * T + n * strips + strip]
// (T = N * strips).  relu_top (may be null): mask by [relu_top > 0].
hipError_t launch_lrn_pool_backward_bf16(const float* pooled, const float* top,
                                         const float* top_diff, const int32_t* mask,
                                         const float* relu_top, uint16_t* Dh, float* sums, int N,
                                         int C, int H, int W, int OH, int OW, int kh, int kw,
                                         int sh, int sw, int ph, int pw, int size, float alpha,
                                         float beta, float k, int Kg, int Kgp, int Ktot, int DHp,
                                         int DWp, int tb, int lb, hipStream_t s,
                                         int mask_u8 = 0);
hipError_t launch_lrn_pool_backward(const float* pooled, const float* top, const float* top_diff,
                                    const int32_t* mask, float* dx, int N, int C, int H, int W,
                                    int OH, int OW, int kh, int kw, int sh, int sw, int ph, int pw,
                                    int size, float alpha, float beta, float k, hipStream_t s,
                                    int mask_u8 = 0);
hipError_t launch_cast_f32_bf16(const float* x, uint16_t* y, int64_t count, hipStream_t s);

// ---- solver (solver.hip)
// Softmax loss forward + backward: per-sample losses, then their fixed-order
// total; prob / diff may be null.
hipError_t launch_softmax_loss(const float* z, const int32_t* labels, int N, int K,
                               float loss_weight, float* loss, float* sample_loss, float* prob,
                               float* diff, hipStream_t s);
// v <- momentum v + lr (g + decay w); w <- w - v (16-byte aligned pointers);
// lr is read from lr_dev when that is non-null.
hipError_t launch_sgd_update(float* w, const float* g, float* v, int64_t count, float lr,
                             const float* lr_dev, float momentum, float decay, hipStream_t s);

}  // namespace caffe_hip
