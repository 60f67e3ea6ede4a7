// qconv_bwd_weight.h -- weight and bias gradients of the quadratic convolution
// layer (arXiv 2204.01701, section 4.3, eq:SD):
//
//   dW_t[o,r,q,c] = sum_{n,i,j} G_t[n,i,j,o] X[n, i*s-p+r, j*s-p+q, c]
//   db_t[o]       = sum_{n,i,j} G_t[n,i,j,o]
//   G_a = G o T_b,  G_b = G o T_a,  G_c = G
//
// ONE implicit GEMM for the three terms, reducing over the output pixels:
//
//   rows    : k' = (r, q, c)           (operand: im2col of X)
//   columns : (t, o), three blocks      (operand: G_t, formed in the prologue)
//   K       : output pixels m = (n, i, j), split over workgroups
//
// Both operands arrive pixel-major (NHWC), so the staging threads load
// PX pixels x VEC channels, form the G_t products in fp32 (accumulating the
// bias sums on the way), transpose the block in registers and write
// pixel-contiguous LDS rows.  Split-K partials go to a workspace and are
// reduced in split order by a second kernel, so the result is deterministic.
#pragma once

#include "qdevice.h"

namespace ql {

struct BwdWeightArgs {
    const void *x, *gy, *ta, *tb;
    float *dw[3];
    float *db[3];
    float *ws_dw;  // [split][3][O][KP]
    float *ws_db;  // [split][3][O]
    int N, H, W, C, O, KH, KW, SH, SW, PH, PW, HO, WO;
    int M, KP;  // M = N*HO*WO output pixels (reduction), KP = KH*KW*C
    int row_tiles, col_tiles, splits, stages_per_split, stages_total;
    int want_db;
    FastDiv fd_howo, fd_wo, fd_c, fd_kw;
};

template <typename T, int BKP, int BO, int WGR, int WGC, int BKB, int PXG, bool VECK>
__global__ __launch_bounds__(kThreads) void qconv_bwd_weight_kernel(const BwdWeightArgs a) {
    constexpr int VEC = Elem<T>::VEC;
    constexpr int ES = (int)sizeof(T);
    constexpr int KE = BKB / ES;    // output pixels per K step
    constexpr int PXX = 16 / ES;    // pixels per X staging job (one 16-byte LDS write per channel)
    constexpr int PITCH = BKB + 16;
    constexpr int ROWS = BKP + 3 * BO;
    constexpr int NKV = BKP / VEC, NOV = BO / VEC;
    constexpr int NJX = NKV * (KE / PXX);  // X jobs: PXX pixels x VEC channels
    constexpr int NJG = NOV * (KE / PXG);  // G jobs: PXG pixels x VEC output channels, three terms
    constexpr int MR = BKP / WGR / 32, MC = BO / WGC / 32;
    static_assert(WGR * WGC == kThreads / 64, "one wave per wave-tile");
    static_assert(NJX + NJG <= kThreads, "one staging job per thread");
    static_assert(PXG * ES == 8 || PXG * ES == 16, "G staging writes 8 or 16 bytes");
    static_assert(MR >= 1 && MC >= 1 && BKB % 32 == 0 && KE % PXX == 0 && KE % PXG == 0, "tile shape");

    __shared__ __attribute__((aligned(16))) char smem[2 * ROWS * PITCH];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wr = wave / WGC, wc = wave % WGC;
    int bid = xcd_remap(blockIdx.x, gridDim.x);
    const int tiles = a.row_tiles * a.col_tiles;
    const int split = bid / tiles;
    bid -= split * tiles;
    const int rt = bid % a.row_tiles, ct = bid / a.row_tiles;
    const int s_begin = split * a.stages_per_split;
    const int s_end = min(s_begin + a.stages_per_split, a.stages_total);
    const bool do_db = a.want_db && rt == 0;

    const T *__restrict__ x = static_cast<const T *>(a.x);
    const T *__restrict__ gy = static_cast<const T *>(a.gy);
    const T *__restrict__ gta = static_cast<const T *>(a.ta);
    const T *__restrict__ gtb = static_cast<const T *>(a.tb);

    const bool is_x = tid < NJX;
    const bool is_g = !is_x && tid < NJX + NJG;
    // X job: channels kv*VEC.. of row tile, pixels pg*PXX.. of each K step.
    const int jx = tid, kv = jx % NKV, pgx = jx / NKV;
    // G job: output channels ov*VEC.., pixels pg*PXG.. of each K step.
    const int jg = tid - NJX, ov = jg % NOV, pgg = jg / NOV;

    // X job geometry (fixed): the VEC rows k' = kbase + e.
    const int kbase = rt * BKP + kv * VEC;
    int xr[VEC], xq[VEC], xc[VEC];
    bool xk[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
        const int kk = VECK ? kbase : kbase + e;  // VECK: one tap for all VEC channels
        const int tap = (int)fdiv((uint32_t)kk, a.fd_c);
        xc[e] = kk - tap * a.C + (VECK ? e : 0);
        xr[e] = (int)fdiv((uint32_t)tap, a.fd_kw);
        xq[e] = tap - xr[e] * a.KW;
        xk[e] = kbase + e < a.KP;
    }
    const int obase = ct * BO + ov * VEC;

    v4u rx[PXX];
    v4u rg[3][PXG];
    float dsum[3][VEC];
#pragma unroll
    for (int t = 0; t < 3; ++t)
#pragma unroll
        for (int e = 0; e < VEC; ++e) dsum[t][e] = 0.0f;

    auto load_stage = [&](int s) {
        if (is_x) {
            const int m0 = s * KE + pgx * PXX;
            int n = (int)fdiv((uint32_t)m0, a.fd_howo);
            const int rem = m0 - n * a.HO * a.WO;
            int oh = (int)fdiv((uint32_t)rem, a.fd_wo);
            int ow = rem - oh * a.WO;
#pragma unroll
            for (int p = 0; p < PXX; ++p) {
                const bool mok = m0 + p < a.M;
                const int ih0 = oh * a.SH - a.PH, iw0 = ow * a.SW - a.PW;
                const size_t nb = (size_t)n * a.H;
                if constexpr (VECK) {
                    const int ih = ih0 + xr[0], iw = iw0 + xq[0];
                    const bool ok = mok && xk[0] && (unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W;
                    rx[p] = ld16(x + ((nb + ih) * a.W + iw) * a.C + xc[0], ok);
                } else {
                    struct alignas(16) V { T e[VEC]; } v;
#pragma unroll
                    for (int e = 0; e < VEC; ++e) {
                        const int ih = ih0 + xr[e], iw = iw0 + xq[e];
                        const bool ok =
                            mok && xk[e] && (unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W;
                        v.e[e] = ok ? x[((nb + ih) * a.W + iw) * a.C + xc[e]] : T(0);
                    }
                    rx[p] = __builtin_bit_cast(v4u, v);
                }
                if (++ow == a.WO) {
                    ow = 0;
                    if (++oh == a.HO) {
                        oh = 0;
                        ++n;
                    }
                }
            }
        } else if (is_g) {
            const int m0 = s * KE + pgg * PXG;
#pragma unroll
            for (int p = 0; p < PXG; ++p) {
                const int m = m0 + p;
                const size_t off = (size_t)m * a.O + obase;
                if constexpr (VECK) {
                    const bool ok = m < a.M && obase < a.O;
                    rg[0][p] = ld16(gy + off, ok);
                    rg[1][p] = ld16(gta + off, ok);
                    rg[2][p] = ld16(gtb + off, ok);
                } else {
                    struct alignas(16) V { T e[VEC]; } v0, v1, v2;
#pragma unroll
                    for (int e = 0; e < VEC; ++e) {
                        const bool ok = m < a.M && obase + e < a.O;
                        v0.e[e] = ok ? gy[off + e] : T(0);
                        v1.e[e] = ok ? gta[off + e] : T(0);
                        v2.e[e] = ok ? gtb[off + e] : T(0);
                    }
                    rg[0][p] = __builtin_bit_cast(v4u, v0);
                    rg[1][p] = __builtin_bit_cast(v4u, v1);
                    rg[2][p] = __builtin_bit_cast(v4u, v2);
                }
            }
        }
    };

    auto store_stage = [&](int b) {
        char *base = smem + b * ROWS * PITCH;
        if (is_x) {
            // PXX pixels x VEC channels -> VEC rows of PXX pixel values (16 bytes each).
#pragma unroll
            for (int e = 0; e < VEC; ++e) {
                uint32_t d[4];
                if constexpr (ES == 2) {
#pragma unroll
                    for (int i = 0; i < 4; ++i) d[i] = vraw<T>(rx[2 * i], e) | (vraw<T>(rx[2 * i + 1], e) << 16);
                } else {
#pragma unroll
                    for (int i = 0; i < 4; ++i) d[i] = vraw<T>(rx[i], e);
                }
                lds_write16(base + (kv * VEC + e) * PITCH + pgx * 16, v4u{d[0], d[1], d[2], d[3]});
            }
        } else if (is_g) {
            // Prologue (eq:SD) in fp32, bias sums, then transpose to pixel-contiguous rows.
            float gv[3][PXG][VEC];
#pragma unroll
            for (int p = 0; p < PXG; ++p)
#pragma unroll
                for (int e = 0; e < VEC; ++e) {
                    const float g = vget<T>(rg[0][p], e);
                    gv[0][p][e] = g * vget<T>(rg[2][p], e);
                    gv[1][p][e] = g * vget<T>(rg[1][p], e);
                    gv[2][p][e] = g;
                }
#pragma unroll
            for (int t = 0; t < 3; ++t)
#pragma unroll
                for (int e = 0; e < VEC; ++e) {
                    float sacc = 0.0f;
#pragma unroll
                    for (int p = 0; p < PXG; ++p) sacc += gv[t][p][e];
                    dsum[t][e] += sacc;
                    char *dst = base + (BKP + t * BO + ov * VEC + e) * PITCH + pgg * PXG * ES;
                    if constexpr (ES == 2) {
                        uint32_t d[PXG / 2];
#pragma unroll
                        for (int i = 0; i < PXG / 2; ++i)
                            d[i] = (t == 2) ? (vraw<T>(rg[0][2 * i], e) | (vraw<T>(rg[0][2 * i + 1], e) << 16))
                                            : pack_bf16x2(gv[t][2 * i][e], gv[t][2 * i + 1][e]);
                        if constexpr (PXG == 4)
                            *reinterpret_cast<v2u *>(dst) = v2u{d[0], d[1]};
                        else
                            lds_write16(dst, v4u{d[0], d[1], d[2], d[3]});
                    } else {
                        uint32_t d[PXG];
#pragma unroll
                        for (int i = 0; i < PXG; ++i) d[i] = __float_as_uint(gv[t][i][e]);
                        if constexpr (PXG == 4)
                            lds_write16(dst, v4u{d[0], d[1], d[2], d[3]});
                        else
                            *reinterpret_cast<v2u *>(dst) = v2u{d[0], d[1]};
                    }
                }
        }
    };

    f32x16_t acc[3][MR][MC];
#pragma unroll
    for (int t = 0; t < 3; ++t)
#pragma unroll
        for (int mr = 0; mr < MR; ++mr)
#pragma unroll
            for (int mc = 0; mc < MC; ++mc)
#pragma unroll
                for (int v = 0; v < 16; ++v) acc[t][mr][mc][v] = 0.0f;

    const int lrow = lane & 31, lhi = lane >> 5;
    auto compute_stage = [&](int b) {
        const char *base = smem + b * ROWS * PITCH;
#pragma unroll
        for (int ch = 0; ch < BKB / 32; ++ch) {
            const int coff = ch * 32 + lhi * 16;
            v4u af[MR];
#pragma unroll
            for (int mr = 0; mr < MR; ++mr)
                af[mr] = lds_read16(base + (wr * (BKP / WGR) + mr * 32 + lrow) * PITCH + coff);
#pragma unroll
            for (int t = 0; t < 3; ++t)
#pragma unroll
                for (int mc = 0; mc < MC; ++mc) {
                    const v4u bf =
                        lds_read16(base + (BKP + t * BO + wc * (BO / WGC) + mc * 32 + lrow) * PITCH + coff);
#pragma unroll
                    for (int mr = 0; mr < MR; ++mr) mfma_chunk<T>(af[mr], bf, acc[t][mr][mc]);
                }
        }
    };

    if (s_begin < s_end) {
        load_stage(s_begin);
        store_stage(0);
        __syncthreads();
        for (int s = s_begin; s < s_end; ++s) {
            const int b = (s - s_begin) & 1;
            const bool more = s + 1 < s_end;
            if (more) load_stage(s + 1);
            compute_stage(b);
            if (more) store_stage(b ^ 1);
            __syncthreads();
        }
    }

    // dW epilogue: rows k', columns o.  Lane holds 4 consecutive k' per group.
    const int krow0 = rt * BKP + wr * (BKP / WGR);
    const int ocol0 = ct * BO + wc * (BO / WGC);
    const bool vec_out = (a.KP & 3) == 0;
#pragma unroll
    for (int t = 0; t < 3; ++t) {
        float *__restrict__ dst =
            a.splits == 1 ? a.dw[t] : a.ws_dw + ((size_t)split * 3 + t) * (size_t)a.O * a.KP;
#pragma unroll
        for (int mr = 0; mr < MR; ++mr)
#pragma unroll
            for (int mc = 0; mc < MC; ++mc) {
                const int o = ocol0 + mc * 32 + lrow;
                if (o >= a.O) continue;
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int k = krow0 + mr * 32 + 8 * g + 4 * lhi;
                    if (k >= a.KP) continue;
                    const size_t off = (size_t)o * a.KP + k;
                    if (vec_out) {
                        store4<float>(dst + off, acc[t][mr][mc][4 * g], acc[t][mr][mc][4 * g + 1],
                                      acc[t][mr][mc][4 * g + 2], acc[t][mr][mc][4 * g + 3]);
                    } else {
#pragma unroll
                        for (int i = 0; i < 4; ++i)
                            if (k + i < a.KP) dst[off + i] = acc[t][mr][mc][4 * g + i];
                    }
                }
            }
    }

    // Bias gradients: the G staging threads hold per-channel sums over their
    // pixels; add them up across the pixel groups in a fixed order.
    if (do_db) {
        constexpr int NPG = KE / PXG;
        float *red = reinterpret_cast<float *>(smem);  // [NPG][3][BO]; LDS is free after the last barrier
        static_assert(NPG * 3 * BO * 4 <= 2 * ROWS * PITCH, "bias scratch fits");
        if (is_g) {
#pragma unroll
            for (int t = 0; t < 3; ++t)
#pragma unroll
                for (int e = 0; e < VEC; ++e) red[(pgg * 3 + t) * BO + ov * VEC + e] = dsum[t][e];
        }
        __syncthreads();
        for (int i = tid; i < 3 * BO; i += kThreads) {
            const int t = i / BO, ol = i % BO;
            const int o = ct * BO + ol;
            if (o >= a.O) continue;
            float s = 0.0f;
            for (int pg = 0; pg < NPG; ++pg) s += red[(pg * 3 + t) * BO + ol];
            if (a.splits == 1)
                a.db[t][o] = s;
            else
                a.ws_db[((size_t)split * 3 + t) * a.O + o] = s;
        }
    }
}

// Split-K reduction of dW_t and db_t partials, in split order.
__global__ __launch_bounds__(kThreads) void qconv_bwd_weight_reduce_kernel(const float *__restrict__ ws_dw,
                                                                           const float *__restrict__ ws_db,
                                                                           int splits, long long ndw, int O,
                                                                           float *dw0, float *dw1, float *dw2,
                                                                           float *db0, float *db1, float *db2,
                                                                           int want_db) {
    const long long total = 3 * ndw + (want_db ? 3LL * O : 0LL);
    for (long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
         idx += (long long)gridDim.x * blockDim.x) {
        if (idx < 3 * ndw) {
            const int t = (int)(idx / ndw);
            const long long i = idx - t * ndw;
            float s = 0.0f;
            for (int sp = 0; sp < splits; ++sp) s += ws_dw[((size_t)sp * 3 + t) * ndw + i];
            float *d = t == 0 ? dw0 : (t == 1 ? dw1 : dw2);
            d[i] = s;
        } else {
            const long long j = idx - 3 * ndw;
            const int t = (int)(j / O), o = (int)(j % O);
            float s = 0.0f;
            for (int sp = 0; sp < splits; ++sp) s += ws_db[((size_t)sp * 3 + t) * O + o];
            float *d = t == 0 ? db0 : (t == 1 ? db1 : db2);
            d[o] = s;
        }
    }
}

}  // namespace ql
