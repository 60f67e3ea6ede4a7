/*
 * qlayer_oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, fp64 direct-summation implementation of the quadratic
 * neuron of QuadraLib (arXiv 2204.01701), used only by the test-suite, by
 * the CPU-baseline leg of the benchmark and by the smoke check to judge the
 * GPU library.  It shares no code, header or constant with the GPU path and
 * must never be linked into, or called from, the product.
 *
 * What it computes (paper section 3.1, equation eq:2ndneuron3):
 *     f(X) = (W_a X) o (W_b X) + (W_c X)
 * where "o" is the Hadamard (elementwise) product (Table 1, note 3).  The
 * neuron is built from three ordinary first-order neurons (section 3.2, P4),
 * so each term carries its own bias, which the equation drops "for
 * simplicity" (Table 1, note 1):
 *     T_t = W_t * X + b_t,   t in {a, b, c}
 *     Y   = T_a o T_b + T_c
 * As a convolution layer "*" is the cross-correlation of a PyTorch
 * nn.Conv2d (section 4.2, encapsulated layer module): zero padding, floor
 * rounding of the output size, dilation 1, groups 1, the same kernel size,
 * stride and padding for all three terms.  As a fully-connected layer
 * (section 3.2, P3) "*" is a matrix-vector product.
 *
 * Backward (section 4.3, equations eq:AD and eq:SD): with G = dl/dY,
 *     G_a = G o T_b,  G_b = G o T_a,  G_c = G            (eq:SD)
 *     dW_t = correlation of G_t with X, db_t = sum of G_t,
 *     dX   = sum over t of the transposed convolution of G_t with W_t.
 *
 * Layouts: activations N x C x H x W, weights O x C x KH x KW (row-major,
 * the logical PyTorch layouts), fp64 throughout.  Bias pointers may be NULL
 * (meaning zero).  Output pointers that are NULL are not written.
 * Parallelised with OpenMP over independent output elements only; no BLAS,
 * no atomics, no blocking or reordering beyond the definition.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define IDX4(a, b, c, d, B, C, D) ((((size_t)(a) * (B) + (b)) * (C) + (c)) * (D) + (d))

static int out_size(int in, int k, int s, int p) { return (in + 2 * p - k) / s + 1; }

int oracle_conv2d_out_size(int in, int k, int s, int p) { return out_size(in, k, s, p); }

/* One first-order term T[n,o,i,j] = b[o] + sum_{c,r,q} W[o,c,r,q] X[n,c,i*s-p+r,j*s-p+q]
 * with zero padding (section 3.2 P4: each term is an ordinary convolution). */
static double conv_term(int C, int H, int W, int KH, int KW, int sh, int sw, int ph, int pw,
                        const double *x, const double *w, const double *b,
                        int n, int o, int i, int j) {
    double acc = b ? b[o] : 0.0;
    for (int c = 0; c < C; ++c)
        for (int r = 0; r < KH; ++r) {
            int ih = i * sh - ph + r;
            if (ih < 0 || ih >= H) continue;
            for (int q = 0; q < KW; ++q) {
                int iw = j * sw - pw + q;
                if (iw < 0 || iw >= W) continue;
                acc += w[IDX4(o, c, r, q, C, KH, KW)] * x[IDX4(n, c, ih, iw, C, H, W)];
            }
        }
    return acc;
}

/* Forward of the quadratic convolution layer (eq:2ndneuron3).  Y, T_a, T_b are
 * N x O x Ho x Wo; any of them may be NULL. */
void oracle_conv2d_fwd(int N, int C, int H, int W, int O, int KH, int KW,
                       int sh, int sw, int ph, int pw,
                       const double *x, const double *wa, const double *wb, const double *wc,
                       const double *ba, const double *bb, const double *bc,
                       double *y, double *ta, double *tb) {
    int Ho = out_size(H, KH, sh, ph), Wo = out_size(W, KW, sw, pw);
    if (Ho < 1 || Wo < 1) return;
    long long total = (long long)N * O * Ho * Wo;
#pragma omp parallel for schedule(static)
    for (long long e = 0; e < total; ++e) {
        int j = (int)(e % Wo), i = (int)((e / Wo) % Ho);
        int o = (int)((e / ((long long)Wo * Ho)) % O), n = (int)(e / ((long long)Wo * Ho * O));
        double Ta = conv_term(C, H, W, KH, KW, sh, sw, ph, pw, x, wa, ba, n, o, i, j);
        double Tb = conv_term(C, H, W, KH, KW, sh, sw, ph, pw, x, wb, bb, n, o, i, j);
        double Tc = conv_term(C, H, W, KH, KW, sh, sw, ph, pw, x, wc, bc, n, o, i, j);
        if (y) y[e] = Ta * Tb + Tc;
        if (ta) ta[e] = Ta;
        if (tb) tb[e] = Tb;
    }
}

/* Backward of the quadratic convolution layer (section 4.3).  The term maps
 * T_a, T_b are regenerated from X and the weights (the hybrid back-propagation
 * of section 4.3 keeps only inputs), then eq:SD gives the per-term output
 * gradients G_a = G o T_b, G_b = G o T_a, G_c = G, and each term's weight,
 * bias and input gradients are those of an ordinary convolution.
 * Any output pointer may be NULL. */
void oracle_conv2d_bwd(int N, int C, int H, int W, int O, int KH, int KW,
                       int sh, int sw, int ph, int pw,
                       const double *x, const double *wa, const double *wb, const double *wc,
                       const double *ba, const double *bb, const double *bc,
                       const double *gy,
                       double *dx, double *dwa, double *dwb, double *dwc,
                       double *dba, double *dbb, double *dbc) {
    int Ho = out_size(H, KH, sh, ph), Wo = out_size(W, KW, sw, pw);
    if (Ho < 1 || Wo < 1) return;
    size_t P = (size_t)N * O * Ho * Wo;
    double *ga = (double *)malloc(P * sizeof(double));
    double *gb = (double *)malloc(P * sizeof(double));
    double *ta = (double *)malloc(P * sizeof(double));
    double *tb = (double *)malloc(P * sizeof(double));
    if (!ga || !gb || !ta || !tb) { free(ga); free(gb); free(ta); free(tb); return; }
    oracle_conv2d_fwd(N, C, H, W, O, KH, KW, sh, sw, ph, pw, x, wa, wb, wc, ba, bb, bc,
                      NULL, ta, tb);
    /* eq:SD: the upstream gradient times the partner term. */
    for (size_t e = 0; e < P; ++e) {
        ga[e] = gy[e] * tb[e];
        gb[e] = gy[e] * ta[e];
    }
    const double *gt[3] = {ga, gb, gy};
    double *dwt[3] = {dwa, dwb, dwc};
    double *dbt[3] = {dba, dbb, dbc};
    const double *wt[3] = {wa, wb, wc};

    /* Weight gradients: dW_t[o,c,r,q] = sum_{n,i,j} G_t[n,o,i,j] X[n,c,i*s-p+r,j*s-p+q]. */
    long long nw = (long long)O * C * KH * KW;
    for (int t = 0; t < 3; ++t) {
        if (!dwt[t]) continue;
        const double *g = gt[t];
        double *dw = dwt[t];
#pragma omp parallel for schedule(static)
        for (long long e = 0; e < nw; ++e) {
            int q = (int)(e % KW), r = (int)((e / KW) % KH);
            int c = (int)((e / ((long long)KW * KH)) % C), o = (int)(e / ((long long)KW * KH * C));
            double acc = 0.0;
            for (int n = 0; n < N; ++n)
                for (int i = 0; i < Ho; ++i) {
                    int ih = i * sh - ph + r;
                    if (ih < 0 || ih >= H) continue;
                    for (int j = 0; j < Wo; ++j) {
                        int iw = j * sw - pw + q;
                        if (iw < 0 || iw >= W) continue;
                        acc += g[IDX4(n, o, i, j, O, Ho, Wo)] * x[IDX4(n, c, ih, iw, C, H, W)];
                    }
                }
            dw[e] = acc;
        }
    }
    /* Bias gradients: db_t[o] = sum_{n,i,j} G_t[n,o,i,j]. */
    for (int t = 0; t < 3; ++t) {
        if (!dbt[t]) continue;
        const double *g = gt[t];
#pragma omp parallel for schedule(static)
        for (int o = 0; o < O; ++o) {
            double acc = 0.0;
            for (int n = 0; n < N; ++n)
                for (int i = 0; i < Ho; ++i)
                    for (int j = 0; j < Wo; ++j) acc += g[IDX4(n, o, i, j, O, Ho, Wo)];
            dbt[t][o] = acc;
        }
    }
    /* Input gradient, gather form: dX[n,c,h,w] = sum_t sum_{o,r,q} G_t[n,o,i,j] W_t[o,c,r,q]
     * over the (i, j) with i*s - p + r = h and j*s - p + q = w. */
    if (dx) {
        long long nx = (long long)N * C * H * W;
#pragma omp parallel for schedule(static)
        for (long long e = 0; e < nx; ++e) {
            int w_ = (int)(e % W), h = (int)((e / W) % H);
            int c = (int)((e / ((long long)W * H)) % C), n = (int)(e / ((long long)W * H * C));
            double acc = 0.0;
            for (int t = 0; t < 3; ++t)
                for (int o = 0; o < O; ++o)
                    for (int r = 0; r < KH; ++r) {
                        int hi = h + ph - r;
                        if (hi < 0 || hi % sh) continue;
                        int i = hi / sh;
                        if (i >= Ho) continue;
                        for (int q = 0; q < KW; ++q) {
                            int wi = w_ + pw - q;
                            if (wi < 0 || wi % sw) continue;
                            int j = wi / sw;
                            if (j >= Wo) continue;
                            acc += gt[t][IDX4(n, o, i, j, O, Ho, Wo)] * wt[t][IDX4(o, c, r, q, C, KH, KW)];
                        }
                    }
            dx[e] = acc;
        }
    }
    free(ga); free(gb); free(ta); free(tb);
}

/* ---------------------------------------------------------------------------
 * The earlier quadratic neuron types the paper compares its design with
 * (Table 1 types and the Table 3 baselines), as convolution layers with the
 * same geometry rules.  neuron: 0 the proposed one (as above), 1 T4, 2 T4 plus
 * identity, 3 T3, 4 T2, 5 T2&4.  With T_t = W_t * X + b_t:
 *   T4:            Y = T_a o T_b
 *   T4 + identity: Y = T_a o T_b + X      (C == O, Ho == H, Wo == W: the
 *                                          shortcut adds input channel o)
 *   T3:            Y = T_a o T_a          (the square of one first-order neuron)
 *   T2:            Y = W_a * (X o X) + b_a (a first-order neuron of the squared input)
 *   T2&4:          Y = T_a o T_b + (W_c * (X o X) + b_c)   (Table 1: the product
 *                  of two first-order terms plus a first-order neuron of the
 *                  squared input; the proposed design is this with X in place
 *                  of X o X in its third term, section 3.1)
 * Unused weights and biases are ignored (may be NULL).  The saved maps:
 * T_a and T_b (T4 types, T2&4), T_a (T3), none (T2).
 * ------------------------------------------------------------------------- */
void oracle_conv2d_fwd_neuron(int neuron, int N, int C, int H, int W, int O, int KH, int KW,
                              int sh, int sw, int ph, int pw,
                              const double *x, const double *wa, const double *wb, const double *wc,
                              const double *ba, const double *bb, const double *bc,
                              double *y, double *ta, double *tb) {
    if (neuron == 0) {
        oracle_conv2d_fwd(N, C, H, W, O, KH, KW, sh, sw, ph, pw, x, wa, wb, wc, ba, bb, bc, y, ta, tb);
        return;
    }
    int Ho = out_size(H, KH, sh, ph), Wo = out_size(W, KW, sw, pw);
    if (Ho < 1 || Wo < 1) return;
    if (neuron == 2 && (C != O || Ho != H || Wo != W)) return;
    size_t nx = (size_t)N * C * H * W;
    double *x2 = NULL;
    if (neuron == 4 || neuron == 5) { /* the squared input, elementwise */
        x2 = (double *)malloc(nx * sizeof(double));
        if (!x2) return;
        for (size_t e = 0; e < nx; ++e) x2[e] = x[e] * x[e];
    }
    long long total = (long long)N * O * Ho * Wo;
#pragma omp parallel for schedule(static)
    for (long long e = 0; e < total; ++e) {
        int j = (int)(e % Wo), i = (int)((e / Wo) % Ho);
        int o = (int)((e / ((long long)Wo * Ho)) % O), n = (int)(e / ((long long)Wo * Ho * O));
        double Ta, Tb = 0.0, out;
        if (neuron == 4) {
            Ta = conv_term(C, H, W, KH, KW, sh, sw, ph, pw, x2, wa, ba, n, o, i, j);
            out = Ta;
        } else {
            Ta = conv_term(C, H, W, KH, KW, sh, sw, ph, pw, x, wa, ba, n, o, i, j);
            if (neuron == 3) {
                out = Ta * Ta;
            } else {
                Tb = conv_term(C, H, W, KH, KW, sh, sw, ph, pw, x, wb, bb, n, o, i, j);
                out = Ta * Tb;
                if (neuron == 2) out += x[IDX4(n, o, i, j, C, H, W)];
                if (neuron == 5) out += conv_term(C, H, W, KH, KW, sh, sw, ph, pw, x2, wc, bc, n, o, i, j);
            }
        }
        if (y) y[e] = out;
        if (ta) ta[e] = Ta;
        if (tb) tb[e] = Tb;
    }
    free(x2);
}

/* Backward of the neuron types above: the per-term output gradients follow
 * from the product rule on each Y,
 *   T4, T4 + identity: G_a = G o T_b, G_b = G o T_a   (plus dX += G for the shortcut)
 *   T3:                G_a = 2 G o T_a
 *   T2:                G_a = G, the operand being X o X, so dW_a correlates G
 *                      with X o X and dX = 2 X o (transposed convolution of G with W_a)
 *   T2&4:              G_a = G o T_b, G_b = G o T_a on the operand X, G_c = G on
 *                      the operand X o X, so dW_c correlates G with X o X and the
 *                      c term's share of dX is 2 X o (transposed convolution of G with W_c)
 * and each term's weight, bias and input gradients are those of an ordinary
 * convolution (the same loops as oracle_conv2d_bwd, written out again here). */
void oracle_conv2d_bwd_neuron(int neuron, int N, int C, int H, int W, int O, int KH, int KW,
                              int sh, int sw, int ph, int pw,
                              const double *x, const double *wa, const double *wb, const double *wc,
                              const double *ba, const double *bb, const double *bc,
                              const double *gy,
                              double *dx, double *dwa, double *dwb, double *dwc,
                              double *dba, double *dbb, double *dbc) {
    if (neuron == 0) {
        oracle_conv2d_bwd(N, C, H, W, O, KH, KW, sh, sw, ph, pw, x, wa, wb, wc, ba, bb, bc, gy,
                          dx, dwa, dwb, dwc, dba, dbb, dbc);
        return;
    }
    int Ho = out_size(H, KH, sh, ph), Wo = out_size(W, KW, sw, pw);
    if (Ho < 1 || Wo < 1) return;
    if (neuron == 2 && (C != O || Ho != H || Wo != W)) return;
    size_t P = (size_t)N * O * Ho * Wo, nx = (size_t)N * C * H * W;
    double *ga = (double *)malloc(P * sizeof(double));
    double *gb = (double *)malloc(P * sizeof(double));
    double *ta = (double *)malloc(P * sizeof(double));
    double *tb = (double *)malloc(P * sizeof(double));
    double *xo = (double *)malloc(nx * sizeof(double)); /* the operand X (or X o X) of terms a, b */
    double *xs = (double *)malloc(nx * sizeof(double)); /* X o X, the operand of T2&4's term c */
    if (!ga || !gb || !ta || !tb || !xo || !xs) {
        free(ga); free(gb); free(ta); free(tb); free(xo); free(xs);
        return;
    }
    oracle_conv2d_fwd_neuron(neuron, N, C, H, W, O, KH, KW, sh, sw, ph, pw, x, wa, wb, wc, ba, bb, bc,
                             NULL, ta, tb);
    int nterm = (neuron == 1 || neuron == 2) ? 2 : (neuron == 5 ? 3 : 1);
    for (size_t e = 0; e < P; ++e) {
        if (nterm >= 2) {
            ga[e] = gy[e] * tb[e];
            gb[e] = gy[e] * ta[e];
        } else if (neuron == 3) {
            ga[e] = 2.0 * gy[e] * ta[e];
        } else {
            ga[e] = gy[e];
        }
    }
    for (size_t e = 0; e < nx; ++e) {
        xo[e] = neuron == 4 ? x[e] * x[e] : x[e];
        xs[e] = x[e] * x[e];
    }
    /* per term: its output gradient, operand, weights and outputs */
    const double *gt[3] = {ga, gb, gy};
    const double *xt[3] = {xo, xo, xs};
    double *dwt[3] = {dwa, dwb, dwc};
    double *dbt[3] = {dba, dbb, dbc};
    const double *wt[3] = {wa, wb, wc};

    long long nw = (long long)O * C * KH * KW;
    for (int t = 0; t < nterm; ++t) {
        if (!dwt[t]) continue;
        const double *g = gt[t], *xx = xt[t];
        double *dw = dwt[t];
#pragma omp parallel for schedule(static)
        for (long long e = 0; e < nw; ++e) {
            int q = (int)(e % KW), r = (int)((e / KW) % KH);
            int c = (int)((e / ((long long)KW * KH)) % C), o = (int)(e / ((long long)KW * KH * C));
            double acc = 0.0;
            for (int n = 0; n < N; ++n)
                for (int i = 0; i < Ho; ++i) {
                    int ih = i * sh - ph + r;
                    if (ih < 0 || ih >= H) continue;
                    for (int j = 0; j < Wo; ++j) {
                        int iw = j * sw - pw + q;
                        if (iw < 0 || iw >= W) continue;
                        acc += g[IDX4(n, o, i, j, O, Ho, Wo)] * xx[IDX4(n, c, ih, iw, C, H, W)];
                    }
                }
            dw[e] = acc;
        }
    }
    for (int t = 0; t < nterm; ++t) {
        if (!dbt[t]) continue;
        const double *g = gt[t];
#pragma omp parallel for schedule(static)
        for (int o = 0; o < O; ++o) {
            double acc = 0.0;
            for (int n = 0; n < N; ++n)
                for (int i = 0; i < Ho; ++i)
                    for (int j = 0; j < Wo; ++j) acc += g[IDX4(n, o, i, j, O, Ho, Wo)];
            dbt[t][o] = acc;
        }
    }
    if (dx) {
        long long nxx = (long long)N * C * H * W;
#pragma omp parallel for schedule(static)
        for (long long e = 0; e < nxx; ++e) {
            int w_ = (int)(e % W), h = (int)((e / W) % H);
            int c = (int)((e / ((long long)W * H)) % C), n = (int)(e / ((long long)W * H * C));
            double part[3] = {0.0, 0.0, 0.0}; /* each term's transposed convolution at (n, c, h, w) */
            for (int t = 0; t < nterm; ++t)
                for (int o = 0; o < O; ++o)
                    for (int r = 0; r < KH; ++r) {
                        int hi = h + ph - r;
                        if (hi < 0 || hi % sh) continue;
                        int i = hi / sh;
                        if (i >= Ho) continue;
                        for (int q = 0; q < KW; ++q) {
                            int wi = w_ + pw - q;
                            if (wi < 0 || wi % sw) continue;
                            int j = wi / sw;
                            if (j >= Wo) continue;
                            part[t] += gt[t][IDX4(n, o, i, j, O, Ho, Wo)] * wt[t][IDX4(o, c, r, q, C, KH, KW)];
                        }
                    }
            double acc;
            if (neuron == 4) acc = part[0] * (2.0 * x[e]);                  /* d(X o X)/dX */
            else if (neuron == 5) acc = part[0] + part[1] + part[2] * (2.0 * x[e]);
            else acc = part[0] + part[1];
            if (neuron == 2) acc += gy[IDX4(n, c, h, w_, O, Ho, Wo)]; /* the identity shortcut */
            dx[e] = acc;
        }
    }
    free(ga); free(gb); free(ta); free(tb); free(xo); free(xs);
}

/* ---------------------------------------------------------------------------
 * Depthwise quadratic convolution (groups = C = O; section 4.2: the layer
 * modules take the depth-wise setting of an ordinary convolution).  Each
 * channel c has its own KH x KW filter per term, W_t[c, r, q], and
 *   T_t[n,c,i,j] = b_t[c] + sum_{r,q} W_t[c,r,q] X[n, c, i*s-p+r, j*s-p+q]
 * with the neuron type's Y as above (the shortcut of T4 + identity needs an
 * unchanged map).  The backward is the same product rule per channel.
 * ------------------------------------------------------------------------- */
static double dw_term(int H, int W, int KH, int KW, int sh, int sw, int ph, int pw, const double *x,
                      const double *w, const double *b, int C, int n, int c, int i, int j) {
    double acc = b ? b[c] : 0.0;
    for (int r = 0; r < KH; ++r) {
        int ih = i * sh - ph + r;
        if (ih < 0 || ih >= H) continue;
        for (int q = 0; q < KW; ++q) {
            int iw = j * sw - pw + q;
            if (iw < 0 || iw >= W) continue;
            acc += w[((size_t)c * KH + r) * KW + q] * x[IDX4(n, c, ih, iw, C, H, W)];
        }
    }
    return acc;
}

void oracle_dwconv2d_fwd(int neuron, int N, int C, int H, int W, int KH, int KW, int sh, int sw, int ph, int pw,
                         const double *x, const double *wa, const double *wb, const double *wc,
                         const double *ba, const double *bb, const double *bc,
                         double *y, double *ta, double *tb) {
    int Ho = out_size(H, KH, sh, ph), Wo = out_size(W, KW, sw, pw);
    if (Ho < 1 || Wo < 1) return;
    if (neuron == 2 && (Ho != H || Wo != W)) return;
    size_t nx = (size_t)N * C * H * W;
    const double *xin = x;
    double *x2 = NULL;
    if (neuron == 4) {
        x2 = (double *)malloc(nx * sizeof(double));
        if (!x2) return;
        for (size_t e = 0; e < nx; ++e) x2[e] = x[e] * x[e];
        xin = x2;
    }
    long long total = (long long)N * C * Ho * Wo;
#pragma omp parallel for schedule(static)
    for (long long e = 0; e < total; ++e) {
        int j = (int)(e % Wo), i = (int)((e / Wo) % Ho);
        int c = (int)((e / ((long long)Wo * Ho)) % C), n = (int)(e / ((long long)Wo * Ho * C));
        double Ta = dw_term(H, W, KH, KW, sh, sw, ph, pw, xin, wa, ba, C, n, c, i, j), Tb = 0.0, out;
        if (neuron == 0 || neuron == 1 || neuron == 2)
            Tb = dw_term(H, W, KH, KW, sh, sw, ph, pw, x, wb, bb, C, n, c, i, j);
        if (neuron == 0) out = Ta * Tb + dw_term(H, W, KH, KW, sh, sw, ph, pw, x, wc, bc, C, n, c, i, j);
        else if (neuron == 1) out = Ta * Tb;
        else if (neuron == 2) out = Ta * Tb + x[IDX4(n, c, i, j, C, H, W)];
        else if (neuron == 3) out = Ta * Ta;
        else out = Ta;
        if (y) y[e] = out;
        if (ta) ta[e] = Ta;
        if (tb) tb[e] = Tb;
    }
    free(x2);
}

void oracle_dwconv2d_bwd(int neuron, int N, int C, int H, int W, int KH, int KW, int sh, int sw, int ph, int pw,
                         const double *x, const double *wa, const double *wb, const double *wc,
                         const double *ba, const double *bb, const double *bc, const double *gy,
                         double *dx, double *dwa, double *dwb, double *dwc,
                         double *dba, double *dbb, double *dbc) {
    int Ho = out_size(H, KH, sh, ph), Wo = out_size(W, KW, sw, pw);
    if (Ho < 1 || Wo < 1) return;
    if (neuron == 2 && (Ho != H || Wo != W)) return;
    size_t P = (size_t)N * C * Ho * Wo, nx = (size_t)N * C * H * W;
    int nterm = neuron == 0 ? 3 : (neuron <= 2 ? 2 : 1);
    double *g3 = (double *)malloc(3 * P * sizeof(double));
    double *ta = (double *)malloc(P * sizeof(double));
    double *tb = (double *)malloc(P * sizeof(double));
    double *xo = (double *)malloc(nx * sizeof(double));
    if (!g3 || !ta || !tb || !xo) { free(g3); free(ta); free(tb); free(xo); return; }
    oracle_dwconv2d_fwd(neuron, N, C, H, W, KH, KW, sh, sw, ph, pw, x, wa, wb, wc, ba, bb, bc, NULL, ta, tb);
    for (size_t e = 0; e < P; ++e) {  /* the per-term output gradients (eq:SD and the types' product rule) */
        if (nterm >= 2) {
            g3[e] = gy[e] * tb[e];
            g3[P + e] = gy[e] * ta[e];
            g3[2 * P + e] = gy[e];
        } else {
            g3[e] = neuron == 3 ? 2.0 * gy[e] * ta[e] : gy[e];
        }
    }
    for (size_t e = 0; e < nx; ++e) xo[e] = neuron == 4 ? x[e] * x[e] : x[e];
    double *dwt[3] = {dwa, dwb, dwc};
    double *dbt[3] = {dba, dbb, dbc};
    const double *wt[3] = {wa, wb, wc};
#pragma omp parallel for schedule(static)
    for (int c = 0; c < C; ++c) {
        for (int t = 0; t < nterm; ++t) {
            const double *g = g3 + (size_t)t * P;
            if (dbt[t]) {
                double acc = 0.0;
                for (int n = 0; n < N; ++n)
                    for (int i = 0; i < Ho; ++i)
                        for (int j = 0; j < Wo; ++j) acc += g[IDX4(n, c, i, j, C, Ho, Wo)];
                dbt[t][c] = acc;
            }
            if (!dwt[t]) continue;
            for (int r = 0; r < KH; ++r)
                for (int q = 0; q < KW; ++q) {
                    double acc = 0.0;
                    for (int n = 0; n < N; ++n)
                        for (int i = 0; i < Ho; ++i) {
                            int ih = i * sh - ph + r;
                            if (ih < 0 || ih >= H) continue;
                            for (int j = 0; j < Wo; ++j) {
                                int iw = j * sw - pw + q;
                                if (iw < 0 || iw >= W) continue;
                                acc += g[IDX4(n, c, i, j, C, Ho, Wo)] * xo[IDX4(n, c, ih, iw, C, H, W)];
                            }
                        }
                    dwt[t][((size_t)c * KH + r) * KW + q] = acc;
                }
        }
    }
    if (dx) {
#pragma omp parallel for schedule(static)
        for (long long e = 0; e < (long long)nx; ++e) {
            int w_ = (int)(e % W), h = (int)((e / W) % H);
            int c = (int)((e / ((long long)W * H)) % C), n = (int)(e / ((long long)W * H * C));
            double acc = 0.0;
            for (int t = 0; t < nterm; ++t)
                for (int r = 0; r < KH; ++r) {
                    int hi = h + ph - r;
                    if (hi < 0 || hi % sh) continue;
                    int i = hi / sh;
                    if (i >= Ho) continue;
                    for (int q = 0; q < KW; ++q) {
                        int wi = w_ + pw - q;
                        if (wi < 0 || wi % sw) continue;
                        int j = wi / sw;
                        if (j >= Wo) continue;
                        acc += g3[(size_t)t * P + IDX4(n, c, i, j, C, Ho, Wo)] * wt[t][((size_t)c * KH + r) * KW + q];
                    }
                }
            if (neuron == 4) acc *= 2.0 * x[e];
            if (neuron == 2) acc += gy[IDX4(n, c, h, w_, C, Ho, Wo)];
            dx[e] = acc;
        }
    }
    free(g3); free(ta); free(tb); free(xo);
}

/* ---------------------------------------------------------------------------
 * Sampled evaluation for full-size checks: the same definitions, evaluated
 * only at requested output positions.
 * ------------------------------------------------------------------------- */

/* Y, T_a, T_b at count positions idx[4*k..4*k+3] = (n, o, i, j). */
void oracle_conv2d_fwd_at(int N, int C, int H, int W, int O, int KH, int KW,
                          int sh, int sw, int ph, int pw,
                          const double *x, const double *wa, const double *wb, const double *wc,
                          const double *ba, const double *bb, const double *bc,
                          long long count, const long long *idx,
                          double *y, double *ta, double *tb) {
    (void)N; (void)O;
#pragma omp parallel for schedule(dynamic, 4)
    for (long long k = 0; k < count; ++k) {
        int n = (int)idx[4 * k], o = (int)idx[4 * k + 1], i = (int)idx[4 * k + 2], j = (int)idx[4 * k + 3];
        double Ta = conv_term(C, H, W, KH, KW, sh, sw, ph, pw, x, wa, ba, n, o, i, j);
        double Tb = conv_term(C, H, W, KH, KW, sh, sw, ph, pw, x, wb, bb, n, o, i, j);
        double Tc = conv_term(C, H, W, KH, KW, sh, sw, ph, pw, x, wc, bc, n, o, i, j);
        if (y) y[k] = Ta * Tb + Tc;
        if (ta) ta[k] = Ta;
        if (tb) tb[k] = Tb;
    }
}

/* dX at count positions idx[4*k..] = (n, c, h, w): the gather form above, with
 * the needed T_a, T_b values regenerated from the definition. */
void oracle_conv2d_dx_at(int N, int C, int H, int W, int O, int KH, int KW,
                         int sh, int sw, int ph, int pw,
                         const double *x, const double *wa, const double *wb, const double *wc,
                         const double *ba, const double *bb, const double *bc,
                         const double *gy, long long count, const long long *idx, double *dx) {
    (void)N; (void)bc;
    int Ho = out_size(H, KH, sh, ph), Wo = out_size(W, KW, sw, pw);
#pragma omp parallel for schedule(dynamic, 1)
    for (long long k = 0; k < count; ++k) {
        int n = (int)idx[4 * k], c = (int)idx[4 * k + 1], h = (int)idx[4 * k + 2], w_ = (int)idx[4 * k + 3];
        double acc = 0.0;
        for (int o = 0; o < O; ++o)
            for (int r = 0; r < KH; ++r) {
                int hi = h + ph - r;
                if (hi < 0 || hi % sh) continue;
                int i = hi / sh;
                if (i >= Ho) continue;
                for (int q = 0; q < KW; ++q) {
                    int wi = w_ + pw - q;
                    if (wi < 0 || wi % sw) continue;
                    int j = wi / sw;
                    if (j >= Wo) continue;
                    double g = gy[IDX4(n, o, i, j, O, Ho, Wo)];
                    double Ta = conv_term(C, H, W, KH, KW, sh, sw, ph, pw, x, wa, ba, n, o, i, j);
                    double Tb = conv_term(C, H, W, KH, KW, sh, sw, ph, pw, x, wb, bb, n, o, i, j);
                    acc += g * Tb * wa[IDX4(o, c, r, q, C, KH, KW)]
                         + g * Ta * wb[IDX4(o, c, r, q, C, KH, KW)]
                         + g * wc[IDX4(o, c, r, q, C, KH, KW)];
                }
            }
        dx[k] = acc;
    }
}

/* dX at every input channel of count input pixels pix[3*k..] = (n, h, w),
 * into dx[k*C + c]: the gather form of oracle_conv2d_dx_at, with T_a and T_b
 * of each output pixel a tap reaches regenerated once and used for all C
 * channels (the same terms added in the same order per element). */
void oracle_conv2d_dx_pixels(int N, int C, int H, int W, int O, int KH, int KW,
                             int sh, int sw, int ph, int pw,
                             const double *x, const double *wa, const double *wb, const double *wc,
                             const double *ba, const double *bb, const double *bc,
                             const double *gy, long long count, const long long *pix, double *dx) {
    (void)N; (void)bc;
    int Ho = out_size(H, KH, sh, ph), Wo = out_size(W, KW, sw, pw);
#pragma omp parallel for schedule(dynamic, 1)
    for (long long k = 0; k < count; ++k) {
        int n = (int)pix[3 * k], h = (int)pix[3 * k + 1], w_ = (int)pix[3 * k + 2];
        double *acc = dx + (size_t)k * C;
        for (int c = 0; c < C; ++c) acc[c] = 0.0;
        for (int o = 0; o < O; ++o)
            for (int r = 0; r < KH; ++r) {
                int hi = h + ph - r;
                if (hi < 0 || hi % sh) continue;
                int i = hi / sh;
                if (i >= Ho) continue;
                for (int q = 0; q < KW; ++q) {
                    int wi = w_ + pw - q;
                    if (wi < 0 || wi % sw) continue;
                    int j = wi / sw;
                    if (j >= Wo) continue;
                    double g = gy[IDX4(n, o, i, j, O, Ho, Wo)];
                    double Ta = conv_term(C, H, W, KH, KW, sh, sw, ph, pw, x, wa, ba, n, o, i, j);
                    double Tb = conv_term(C, H, W, KH, KW, sh, sw, ph, pw, x, wb, bb, n, o, i, j);
                    for (int c = 0; c < C; ++c)
                        acc[c] += g * Tb * wa[IDX4(o, c, r, q, C, KH, KW)]
                                + g * Ta * wb[IDX4(o, c, r, q, C, KH, KW)]
                                + g * wc[IDX4(o, c, r, q, C, KH, KW)];
                }
            }
    }
}

/* Weight and bias gradients of one output channel o: dW_t[o,:,:,:] (C*KH*KW
 * values each) and db_t[o].  Any output pointer may be NULL. */
void oracle_conv2d_dw_channel(int N, int C, int H, int W, int O, int KH, int KW,
                              int sh, int sw, int ph, int pw,
                              const double *x, const double *wa, const double *wb, const double *wc,
                              const double *ba, const double *bb, const double *bc,
                              const double *gy, int o,
                              double *dwa, double *dwb, double *dwc,
                              double *dba, double *dbb, double *dbc) {
    (void)wc; (void)bc;
    int Ho = out_size(H, KH, sh, ph), Wo = out_size(W, KW, sw, pw);
    size_t S = (size_t)N * Ho * Wo;
    double *ga = (double *)malloc(S * sizeof(double));
    double *gb = (double *)malloc(S * sizeof(double));
    double *gc = (double *)malloc(S * sizeof(double));
    if (!ga || !gb || !gc) { free(ga); free(gb); free(gc); return; }
#pragma omp parallel for schedule(static)
    for (long long e = 0; e < (long long)S; ++e) {
        int j = (int)(e % Wo), i = (int)((e / Wo) % Ho), n = (int)(e / ((long long)Wo * Ho));
        double g = gy[IDX4(n, o, i, j, O, Ho, Wo)];
        double Ta = conv_term(C, H, W, KH, KW, sh, sw, ph, pw, x, wa, ba, n, o, i, j);
        double Tb = conv_term(C, H, W, KH, KW, sh, sw, ph, pw, x, wb, bb, n, o, i, j);
        ga[e] = g * Tb;
        gb[e] = g * Ta;
        gc[e] = g;
    }
    const double *gt[3] = {ga, gb, gc};
    double *dwt[3] = {dwa, dwb, dwc};
    double *dbt[3] = {dba, dbb, dbc};
    long long nk = (long long)C * KH * KW;
    for (int t = 0; t < 3; ++t) {
        if (dwt[t]) {
            const double *g = gt[t];
            double *dw = dwt[t];
#pragma omp parallel for schedule(static)
            for (long long e = 0; e < nk; ++e) {
                int q = (int)(e % KW), r = (int)((e / KW) % KH), c = (int)(e / ((long long)KW * KH));
                double acc = 0.0;
                for (int n = 0; n < N; ++n)
                    for (int i = 0; i < Ho; ++i) {
                        int ih = i * sh - ph + r;
                        if (ih < 0 || ih >= H) continue;
                        for (int j = 0; j < Wo; ++j) {
                            int iw = j * sw - pw + q;
                            if (iw < 0 || iw >= W) continue;
                            acc += g[((size_t)n * Ho + i) * Wo + j] * x[IDX4(n, c, ih, iw, C, H, W)];
                        }
                    }
                dw[e] = acc;
            }
        }
        if (dbt[t]) {
            double acc = 0.0;
            for (size_t e = 0; e < S; ++e) acc += gt[t][e];
            dbt[t][0] = acc;
        }
    }
    free(ga); free(gb); free(gc);
}

/* ---------------------------------------------------------------------------
 * Fully-connected quadratic layer (section 3.2 P3):
 *     T_t = X W_t^T + b_t,  Y = T_a o T_b + T_c
 * X is B x I, W_t is O x I, Y, T_t are B x O.  Written directly, not through
 * the convolution code, so the two can be checked against each other.
 * ------------------------------------------------------------------------- */
static double fc_term(int I, const double *x, const double *w, const double *b, int row, int o) {
    double acc = b ? b[o] : 0.0;
    for (int k = 0; k < I; ++k) acc += x[(size_t)row * I + k] * w[(size_t)o * I + k];
    return acc;
}

void oracle_linear_fwd(int B, int I, int O,
                       const double *x, const double *wa, const double *wb, const double *wc,
                       const double *ba, const double *bb, const double *bc,
                       double *y, double *ta, double *tb) {
    long long total = (long long)B * O;
#pragma omp parallel for schedule(static)
    for (long long e = 0; e < total; ++e) {
        int row = (int)(e / O), o = (int)(e % O);
        double Ta = fc_term(I, x, wa, ba, row, o);
        double Tb = fc_term(I, x, wb, bb, row, o);
        double Tc = fc_term(I, x, wc, bc, row, o);
        if (y) y[e] = Ta * Tb + Tc;
        if (ta) ta[e] = Ta;
        if (tb) tb[e] = Tb;
    }
}

/* Backward of the fully-connected layer: G_a = G o T_b, G_b = G o T_a, G_c = G
 * (eq:SD); dW_t = G_t^T X; db_t = column sums of G_t; dX = sum_t G_t W_t. */
void oracle_linear_bwd(int B, int I, int O,
                       const double *x, const double *wa, const double *wb, const double *wc,
                       const double *ba, const double *bb, const double *bc,
                       const double *gy,
                       double *dx, double *dwa, double *dwb, double *dwc,
                       double *dba, double *dbb, double *dbc) {
    size_t P = (size_t)B * O;
    double *ga = (double *)malloc(P * sizeof(double));
    double *gb = (double *)malloc(P * sizeof(double));
    if (!ga || !gb) { free(ga); free(gb); return; }
#pragma omp parallel for schedule(static)
    for (long long e = 0; e < (long long)P; ++e) {
        int row = (int)(e / O), o = (int)(e % O);
        double Ta = fc_term(I, x, wa, ba, row, o);
        double Tb = fc_term(I, x, wb, bb, row, o);
        ga[e] = gy[e] * Tb;
        gb[e] = gy[e] * Ta;
    }
    const double *gt[3] = {ga, gb, gy};
    const double *wt[3] = {wa, wb, wc};
    double *dwt[3] = {dwa, dwb, dwc};
    double *dbt[3] = {dba, dbb, dbc};
    for (int t = 0; t < 3; ++t) {
        if (dwt[t]) {
#pragma omp parallel for schedule(static)
            for (long long e = 0; e < (long long)O * I; ++e) {
                int o = (int)(e / I), k = (int)(e % I);
                double acc = 0.0;
                for (int row = 0; row < B; ++row) acc += gt[t][(size_t)row * O + o] * x[(size_t)row * I + k];
                dwt[t][e] = acc;
            }
        }
        if (dbt[t]) {
#pragma omp parallel for schedule(static)
            for (int o = 0; o < O; ++o) {
                double acc = 0.0;
                for (int row = 0; row < B; ++row) acc += gt[t][(size_t)row * O + o];
                dbt[t][o] = acc;
            }
        }
    }
    if (dx) {
#pragma omp parallel for schedule(static)
        for (long long e = 0; e < (long long)B * I; ++e) {
            int row = (int)(e / I), k = (int)(e % I);
            double acc = 0.0;
            for (int t = 0; t < 3; ++t)
                for (int o = 0; o < O; ++o) acc += gt[t][(size_t)row * O + o] * wt[t][(size_t)o * I + k];
            dx[e] = acc;
        }
    }
    free(ga); free(gb);
}

/* Sampled FC forward: idx[2*k..] = (row, o). */
void oracle_linear_fwd_at(int B, int I, int O,
                          const double *x, const double *wa, const double *wb, const double *wc,
                          const double *ba, const double *bb, const double *bc,
                          long long count, const long long *idx,
                          double *y, double *ta, double *tb) {
    (void)B; (void)O;
#pragma omp parallel for schedule(static)
    for (long long k = 0; k < count; ++k) {
        int row = (int)idx[2 * k], o = (int)idx[2 * k + 1];
        double Ta = fc_term(I, x, wa, ba, row, o);
        double Tb = fc_term(I, x, wb, bb, row, o);
        double Tc = fc_term(I, x, wc, bc, row, o);
        if (y) y[k] = Ta * Tb + Tc;
        if (ta) ta[k] = Ta;
        if (tb) tb[k] = Tb;
    }
}

/* Sampled FC input gradient: dX[row, :] for each requested row (I values each). */
void oracle_linear_dx_rows(int B, int I, int O,
                           const double *x, const double *wa, const double *wb, const double *wc,
                           const double *ba, const double *bb, const double *bc,
                           const double *gy, long long count, const long long *rows, double *dx) {
    (void)B; (void)bc;
    for (long long k = 0; k < count; ++k) {
        int row = (int)rows[k];
        double *ga = (double *)malloc((size_t)O * sizeof(double));
        double *gb = (double *)malloc((size_t)O * sizeof(double));
        if (!ga || !gb) { free(ga); free(gb); return; }
#pragma omp parallel for schedule(static)
        for (int o = 0; o < O; ++o) {
            double g = gy[(size_t)row * O + o];
            ga[o] = g * fc_term(I, x, wb, bb, row, o);
            gb[o] = g * fc_term(I, x, wa, ba, row, o);
        }
#pragma omp parallel for schedule(static)
        for (int i = 0; i < I; ++i) {
            double acc = 0.0;
            for (int o = 0; o < O; ++o)
                acc += ga[o] * wa[(size_t)o * I + i] + gb[o] * wb[(size_t)o * I + i]
                     + gy[(size_t)row * O + o] * wc[(size_t)o * I + i];
            dx[(size_t)k * I + i] = acc;
        }
        free(ga); free(gb);
    }
}

/* Sampled FC weight/bias gradients of one output unit o: dW_t[o, :] (I values)
 * and db_t[o]. */
void oracle_linear_dw_row(int B, int I, int O,
                          const double *x, const double *wa, const double *wb, const double *wc,
                          const double *ba, const double *bb, const double *bc,
                          const double *gy, int o,
                          double *dwa, double *dwb, double *dwc,
                          double *dba, double *dbb, double *dbc) {
    (void)wc; (void)bc;
    double *ga = (double *)malloc((size_t)B * sizeof(double));
    double *gb = (double *)malloc((size_t)B * sizeof(double));
    if (!ga || !gb) { free(ga); free(gb); return; }
#pragma omp parallel for schedule(static)
    for (int row = 0; row < B; ++row) {
        double g = gy[(size_t)row * O + o];
        ga[row] = g * fc_term(I, x, wb, bb, row, o);
        gb[row] = g * fc_term(I, x, wa, ba, row, o);
    }
#pragma omp parallel for schedule(static)
    for (int i = 0; i < I; ++i) {
        double sa = 0.0, sb = 0.0, sc = 0.0;
        for (int row = 0; row < B; ++row) {
            double xv = x[(size_t)row * I + i];
            sa += ga[row] * xv;
            sb += gb[row] * xv;
            sc += gy[(size_t)row * O + o] * xv;
        }
        if (dwa) dwa[i] = sa;
        if (dwb) dwb[i] = sb;
        if (dwc) dwc[i] = sc;
    }
    double sa = 0.0, sb = 0.0, sc = 0.0;
    for (int row = 0; row < B; ++row) {
        sa += ga[row]; sb += gb[row]; sc += gy[(size_t)row * O + o];
    }
    if (dba) *dba = sa;
    if (dbb) *dbb = sb;
    if (dbc) *dbc = sc;
    free(ga); free(gb);
}

/* ------------------------------------------------------------------------
 * Forward epilogue of a layer output (section 4.2, model construction:
 * batch normalization regulates the quadratic layers' output values, and
 * deeper networks put an activation after them).  y is N x O x P (P = Ho*Wo;
 * a dense output has P = 1).  Per channel o, with optional scale/shift
 * (a batch normalization with fixed statistics folded to y' = s y + t) and
 * an optional ReLU:
 *     y'[n,o,p] = relu(scale[o] * y[n,o,p] + shift[o])
 * and the statistics a training-mode batch normalization of y' needs:
 *     sum[o] = sum_{n,p} y'[n,o,p],   sumsq[o] = sum_{n,p} y'[n,o,p]^2
 * ------------------------------------------------------------------------ */
void oracle_epilogue(int N, int O, long long P, const double *y, const double *scale, const double *shift, int relu,
                     double *yo, double *sum, double *sumsq) {
#pragma omp parallel for schedule(static)
    for (int o = 0; o < O; ++o) {
        double s = 0.0, s2 = 0.0;
        for (int n = 0; n < N; ++n) {
            for (long long p = 0; p < P; ++p) {
                size_t i = ((size_t)n * O + o) * (size_t)P + (size_t)p;
                double v = y[i];
                if (scale) v = scale[o] * v;
                if (shift) v = v + shift[o];
                if (relu && v < 0.0) v = 0.0;
                yo[i] = v;
                s += v;
                s2 += v * v;
            }
        }
        sum[o] = s;
        sumsq[o] = s2;
    }
}
