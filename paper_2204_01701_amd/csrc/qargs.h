// qargs.h -- kernel argument blocks (passed by value) of the quadratic-layer kernels.
#pragma once

#include "qfastdiv.h"

namespace ql {

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
    FastDiv fd_howo, fd_wo, fd_c, fd_kw;
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
    FastDiv fd_hw, fd_w, fd_o, fd_kw, fd_sh, fd_sw;
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
    FastDiv fd_howo, fd_wo, fd_c, fd_kw;
};

}  // namespace ql
