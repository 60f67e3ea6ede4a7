// qargs.h -- kernel argument blocks (passed by value) of the quadratic-layer kernels.
#pragma once

#include <hip/hip_runtime.h>

#include "qfastdiv.h"

namespace ql {

// Neuron types (arXiv 2204.01701: the proposed design, section 3.1, and the
// earlier ones of Table 1 that Table 3 compares against), with T_t = W_t X + b_t:
//   NEURON_QUADRA  Y = T_a o T_b + T_c      NEURON_T4  Y = T_a o T_b
//   NEURON_T4I     Y = T_a o T_b + X        NEURON_T3  Y = T_a o T_a
//   NEURON_T2      Y = W_a (X o X) + b_a
//   NEURON_T24     Y = T_a o T_b + W_c (X o X) + b_c   (T2&4 of Table 1)
enum { NEURON_QUADRA = 0, NEURON_T4 = 1, NEURON_T4I = 2, NEURON_T3 = 3, NEURON_T2 = 4, NEURON_T24 = 5 };
// The kernels' compile-time operand mode: which first-order terms exist and
// what feeds them.  OM_PAIR covers T4 and T4 + identity (they differ only in
// the epilogue, a run-time switch).  OM_QSQ is the three-term layout of
// OM_QUADRA whose third term sees X o X: the pixel operand of that term's
// MFMAs is squared in registers (forward: the X tile, weight gradient: the
// X rows), and its share of the input gradient is accumulated apart and
// multiplied by 2 X in the epilogue.
enum { OM_QUADRA = 0, OM_PAIR = 1, OM_SQUARE = 2, OM_SQIN = 3, OM_QSQ = 4 };
__host__ __device__ constexpr int om_of_neuron(int ne) {
    return ne == NEURON_QUADRA ? OM_QUADRA
                               : (ne == NEURON_T24 ? OM_QSQ
                                                   : (ne <= NEURON_T4I ? OM_PAIR : (ne == NEURON_T3 ? OM_SQUARE : OM_SQIN)));
}
// first-order terms (weights) of a mode
__host__ __device__ constexpr int om_terms(int om) {
    return (om == OM_QUADRA || om == OM_QSQ) ? 3 : (om == OM_PAIR ? 2 : 1);
}
// output-side maps the backward stages: G, T_a, T_b / G, T_a / G
__host__ __device__ constexpr int om_gmaps(int om) { return om == OM_SQIN ? 1 : (om == OM_SQUARE ? 2 : 3); }
// the modes whose backward operands are G o T_b, G o T_a, G (the proposed neuron's)
__host__ __device__ constexpr bool om_three(int om) { return om == OM_QUADRA || om == OM_QSQ; }

// Forward epilogue of the layer output (section 4.2, model construction:
// batch normalization after the quadratic layers, an activation in deeper
// networks): y' = relu(scale[o] y + shift[o]) per output channel o (a batch
// normalization with fixed statistics folded to scale and shift), stored in
// place of y; the per-channel sums of y' and y'^2 (training-mode statistics)
// are gathered from the stored values.
struct EpiArgs {
    const float *scale, *shift;  // per output channel, or NULL (1 and 0)
    int relu;
};

// Whether the forward kernel of a tile configuration writes its output tiles
// through the LDS ring (the path that also gathers the epilogue statistics):
// one staged map of BCOL pixel rows of BR channels (padded by 16 bytes) fits
// the ring of NS stages of 3 BR + BCOL 64-byte rows.
__host__ __device__ constexpr bool fwd_staged_fits(int BR, int BCOL, int NS, int E) {
    return BCOL * (BR * E + 16) <= NS * (3 * BR + BCOL) * 64;
}

// Forward: ONE implicit GEMM, rows = output channels (three term blocks
// W_a | W_b | W_c), columns = output pixels, K = (r, q, c).
struct FwdArgs {
    const void *x;
    const void *w[3];
    const float *bias[3];
    void *y, *ta, *tb;
    float *ws;  // split-K partials [split][3][M][O]
    const void *zero;  // 16 zero bytes: the source of masked-off DMA lanes
    int N, H, W, C, O, KH, KW, SH, SW, PH, PW, HO, WO;
    int M, K;  // GEMM extents: M = N*HO*WO pixels, K = KH*KW*C
    int row_tiles, col_tiles, splits, stages_per_split, stages_total;
    int neuron;  // NEURON_*: the epilogue (T4 + identity reads X at the output pixel)
    int xsq;     // T2: x already holds X o X (squared by a pre-pass), no squaring in the kernel
    EpiArgs epi;
    float *stat_part;  // staged epilogue: per pixel tile ct, partial sums of y' [ct][O] and y'^2 [ct][O]; or NULL
    // Position-major pixel order (channel-aligned kernels only): GEMM column m
    // is output position m / N of image m % N, stored at NHWC row
    // (m % N) HO WO + m / N.  A pixel tile then spans few positions, and the K
    // steps of taps that lie in the zero padding for all of them are skipped:
    // the K range is the tile's in-bounds taps, cps = C / KE steps each.
    int pm, cps;
    FastDiv fd_howo, fd_wo, fd_c, fd_kw, fd_n, fd_cps;
};

// Input gradient: rows = input channels, columns = input pixels,
// K = (t, r, q, o) with the per-term weights pre-transposed to C x KH x KW x O.
struct BwdDataArgs {
    const void *gy, *ta, *tb;
    const void *wt[3];  // per-term weights transposed to C x KH x KW x O
    void *dx;
    float *ws;  // split-K partials [split][M][C]
    const void *zero;
    int N, H, W, C, O, KH, KW, SH, SW, PH, PW, HO, WO;
    int M, K;  // M = N*H*W input pixels, K = KH*KW*O per term
    int row_tiles, col_tiles, splits, stages_per_split, stages_total;
    int neuron;       // NEURON_*: the epilogue adds G (T4 + identity) or multiplies by 2 X (T2)
    const void *xin;  // X (N x H x W x C) for T2, else unused
    // Position-major pixel order (channel-aligned kernels, the proposed neuron
    // only): GEMM column m is input position m / N of image m % N, at NHWC row
    // (m % N) H W + m / N; a tile's K range is the taps whose output pixel lies
    // in the map for some position of the tile, ops = O / KE steps each.
    int pm, ops;
    int order;  // block order of the split-K grid (tile_coord)
    FastDiv fd_hw, fd_w, fd_o, fd_kw, fd_sh, fd_sw, fd_n, fd_ops;
};

// Weight/bias gradients: rows = k' = (r, q, c), columns = (t, o), K = output pixels.
struct BwdWeightArgs {
    const void *x, *gy, *ta, *tb;
    float *dw[3];
    float *db[3];
    float *ws_dw;  // [split][3][O][KP]
    float *ws_db;  // [split][3][O]
    const void *zero;
    int N, H, W, C, O, KH, KW, SH, SW, PH, PW, HO, WO;
    int M, KP;  // M = N*HO*WO output pixels (reduction), KP = KH*KW*C
    int row_tiles, col_tiles, splits, stages_per_split, stages_total;
    int want_db;
    int C_out;  // channels of dW_t as stored (< C when X arrives zero-padded to C channels)
    // Stride 1 with HO == H, WO == W: the X address of pixel m at a fixed tap is
    // linear in m, and a K step advances each lane's (oh, ow) by lin_dq rows
    // (mod HO) and lin_dr columns, with one carry.
    int lin, lin_dq, lin_dr;
    int neuron;
    FastDiv fd_howo, fd_wo, fd_c, fd_kw;
};

}  // namespace ql
