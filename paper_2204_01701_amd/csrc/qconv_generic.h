// qconv_generic.h -- register-staged kernels of the quadratic layer for the
// shapes the pipelined kernels do not take (channel counts that are not a
// multiple of the 16-byte vector, e.g. 3-channel image inputs) and for the
// fp32 weight gradient.
//
// Forward (arXiv 2204.01701, section 3.1 eq:2ndneuron3): one implicit GEMM
// for the three terms with the product and sum in the accumulator epilogue.
// Input gradient (section 4.3 eq:AD / eq:SD): one implicit GEMM over
// (t, r, q, o) with G_a = G o T_b, G_b = G o T_a, G_c = G formed while staging.
// Weight/bias gradients (eq:SD): one implicit GEMM over the output pixels with
// the products formed, bias sums accumulated and the block transposed while
// staging.  Each K step is loaded into registers one step ahead and written
// to padded LDS rows.
#pragma once

#include "qargs.h"
#include "qdevice.h"

namespace ql {

// OM (qargs.h): the neuron type's terms; T2 squares the pixel operand while staging.
template <typename T, int BR, int BCOL, int WGR, int WGC, int BKB, bool VECK, int OM = OM_QUADRA>
__global__ __launch_bounds__(kThreads) void qconv_fwd_generic_kernel(const FwdArgs a) {
    constexpr int VEC = Elem<T>::VEC;
    constexpr int NTM = om_terms(OM);
    constexpr int NB = BKB / 16;  // 16-byte vectors per row per K step
    constexpr int KE = NB * VEC;  // reduction elements per K step
    constexpr int PITCH = BKB + 16;
    constexpr int ROWS = 3 * BR + BCOL;
    constexpr int RSTEP = kThreads / NB;          // rows covered by one pass of the workgroup
    constexpr int NVT = BR * NB / kThreads;       // weight vectors per thread per term
    constexpr int NVP = BCOL * NB / kThreads;     // pixel vectors per thread
    constexpr int MR = BR / WGR / 32, MC = BCOL / WGC / 32;
    static_assert(WGR * WGC == kThreads / 64, "one wave per wave-tile");
    static_assert((BR * NB) % kThreads == 0 && (BCOL * NB) % kThreads == 0, "even load split");
    static_assert(MR >= 1 && MC >= 1 && BKB % 32 == 0, "tile shape");

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

    const T *__restrict__ x = static_cast<const T *>(a.x);
    const T *__restrict__ w0 = static_cast<const T *>(a.w[0]);
    const T *__restrict__ w1 = static_cast<const T *>(a.w[1]);
    const T *__restrict__ w2 = static_cast<const T *>(a.w[2]);

    const int c16 = tid % NB;
    const int rsub = tid / NB;

    // Load descriptors, fixed for the whole K loop.
    int woff[NVT];
#pragma unroll
    for (int j = 0; j < NVT; ++j) {
        const int o = rt * BR + rsub + j * RSTEP;
        woff[j] = (o < a.O) ? o * a.K : -1;
    }
    int xoff[NVP], ih0[NVP], iw0[NVP];
#pragma unroll
    for (int j = 0; j < NVP; ++j) {
        const int m = ct * BCOL + rsub + j * RSTEP;
        if (m < a.M) {
            const int n = (int)fdiv((uint32_t)m, a.fd_howo);
            const int rem = m - n * a.HO * a.WO;
            const int oh = (int)fdiv((uint32_t)rem, a.fd_wo);
            const int ow = rem - oh * a.WO;
            xoff[j] = n * a.H * a.W * a.C;
            ih0[j] = oh * a.SH - a.PH;
            iw0[j] = ow * a.SW - a.PW;
        } else {
            xoff[j] = -1;
            ih0[j] = 0;
            iw0[j] = 0;
        }
    }

    v4u rw[NTM][NVT], rx[NVP];

    auto load_stage = [&](int s) {
        const int k = s * KE + c16 * VEC;
        if constexpr (VECK) {
            // C % VEC == 0: the VEC elements share one tap (r, q).
            const bool kin = k < a.K;
            const int tap = (int)fdiv((uint32_t)k, a.fd_c);
            const int c = k - tap * a.C;
            const int r = (int)fdiv((uint32_t)tap, a.fd_kw);
            const int q = tap - r * a.KW;
#pragma unroll
            for (int j = 0; j < NVT; ++j) {
                const bool ok = kin && woff[j] >= 0;
                rw[0][j] = ld16(w0 + woff[j] + k, ok);
                if constexpr (NTM >= 2) rw[1][j] = ld16(w1 + woff[j] + k, ok);
                if constexpr (NTM >= 3) rw[2][j] = ld16(w2 + woff[j] + k, ok);
            }
#pragma unroll
            for (int j = 0; j < NVP; ++j) {
                const int ih = ih0[j] + r, iw = iw0[j] + q;
                const bool ok = kin && xoff[j] >= 0 && (unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W;
                rx[j] = ld16(x + xoff[j] + (ih * a.W + iw) * a.C + c, ok);
            }
        } else {
            // General C: every element decodes its own (r, q, c).
            struct alignas(16) V { T e[VEC]; };
            V vw[NTM][NVT], vx[NVP];
#pragma unroll
            for (int e = 0; e < VEC; ++e) {
                const int ke = k + e;
                const bool kin = ke < a.K;
                const int tap = (int)fdiv((uint32_t)ke, a.fd_c);
                const int c = ke - tap * a.C;
                const int r = (int)fdiv((uint32_t)tap, a.fd_kw);
                const int q = tap - r * a.KW;
#pragma unroll
                for (int j = 0; j < NVT; ++j) {
                    const bool ok = kin && woff[j] >= 0;
                    vw[0][j].e[e] = ok ? w0[woff[j] + ke] : T(0);
                    if constexpr (NTM >= 2) vw[1][j].e[e] = ok ? w1[woff[j] + ke] : T(0);
                    if constexpr (NTM >= 3) vw[2][j].e[e] = ok ? w2[woff[j] + ke] : T(0);
                }
#pragma unroll
                for (int j = 0; j < NVP; ++j) {
                    const int ih = ih0[j] + r, iw = iw0[j] + q;
                    const bool ok =
                        kin && xoff[j] >= 0 && (unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W;
                    vx[j].e[e] = ok ? x[xoff[j] + (ih * a.W + iw) * a.C + c] : T(0);
                }
            }
#pragma unroll
            for (int j = 0; j < NVT; ++j)
#pragma unroll
                for (int t = 0; t < NTM; ++t) rw[t][j] = __builtin_bit_cast(v4u, vw[t][j]);
#pragma unroll
            for (int j = 0; j < NVP; ++j) rx[j] = __builtin_bit_cast(v4u, vx[j]);
        }
        if constexpr (OM == OM_SQIN) {
            if (!a.xsq) {
#pragma unroll
                for (int j = 0; j < NVP; ++j) rx[j] = square_frag<T>(rx[j]);
            }
        }
    };

    auto store_stage = [&](int b) {
        char *base = smem + b * ROWS * PITCH;
#pragma unroll
        for (int t = 0; t < NTM; ++t)
#pragma unroll
            for (int j = 0; j < NVT; ++j)
                lds_write16(base + (t * BR + rsub + j * RSTEP) * PITCH + c16 * 16, rw[t][j]);
#pragma unroll
        for (int j = 0; j < NVP; ++j)
            lds_write16(base + (3 * BR + rsub + j * RSTEP) * PITCH + c16 * 16, rx[j]);
    };

    // Accumulators; the biases are preloaded when the whole K range is ours.
    f32x16_t acc[NTM][MR][MC];
    const int lrow = lane & 31, lhi = lane >> 5;
    const int orow0 = rt * BR + wr * (BR / WGR);
#pragma unroll
    for (int t = 0; t < NTM; ++t) {
        const float *bp = a.bias[t];
#pragma unroll
        for (int mr = 0; mr < MR; ++mr) {
            f32x16_t init;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int o = orow0 + mr * 32 + 8 * (v >> 2) + 4 * lhi + (v & 3);
                init[v] = (a.splits == 1 && bp != nullptr && o < a.O) ? bp[o] : 0.0f;
            }
#pragma unroll
            for (int mc = 0; mc < MC; ++mc) acc[t][mr][mc] = init;
        }
    }

    auto compute_stage = [&](int b) {
        const char *base = smem + b * ROWS * PITCH;
#pragma unroll
        for (int ch = 0; ch < BKB / 32; ++ch) {
            const int coff = ch * 32 + lhi * 16;
            v4u bf[MC];
#pragma unroll
            for (int mc = 0; mc < MC; ++mc)
                bf[mc] = lds_read16(base + (3 * BR + wc * (BCOL / WGC) + mc * 32 + lrow) * PITCH + coff);
            v4u bsq[MC];  // T2&4: the third term's pixel operand X o X
            if constexpr (OM == OM_QSQ) {
#pragma unroll
                for (int mc = 0; mc < MC; ++mc) bsq[mc] = square_frag<T>(bf[mc]);
            }
#pragma unroll
            for (int t = 0; t < NTM; ++t)
#pragma unroll
                for (int mr = 0; mr < MR; ++mr) {
                    const v4u af = lds_read16(base + (t * BR + wr * (BR / WGR) + mr * 32 + lrow) * PITCH + coff);
#pragma unroll
                    for (int mc = 0; mc < MC; ++mc)
                        mfma_chunk<T>(af, (OM == OM_QSQ && t == 2) ? bsq[mc] : bf[mc], acc[t][mr][mc]);
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

    // Epilogue: the neuron type's Y (j = 0) and the saved maps T_a, T_b (j = 1, 2).
    auto outv = [&](int j, int mr, int mc, int v, float xs) -> float {
        const float fa = acc[0][mr][mc][v];
        if (j == 1) return fa;
        if constexpr (om_three(OM) || OM == OM_PAIR) {
            const float fb = acc[1][mr][mc][v];
            if (j == 2) return fb;
            if constexpr (om_three(OM)) return fa * fb + acc[2][mr][mc][v];
            else return fa * fb + xs;
        } else if constexpr (OM == OM_SQUARE) {
            return fa * fa;
        } else {
            return fa;
        }
    };
    const bool shortcut = OM == OM_PAIR && a.neuron == NEURON_T4I;  // C == O: X at the output pixel
    const int pcol0 = ct * BCOL + wc * (BCOL / WGC);
    const bool vec_out = (a.O & 3) == 0;
    if (a.splits == 1) {
        T *__restrict__ y = static_cast<T *>(a.y);
        T *__restrict__ ta = static_cast<T *>(a.ta);
        T *__restrict__ tb = NTM >= 2 ? static_cast<T *>(a.tb) : nullptr;
#pragma unroll
        for (int mr = 0; mr < MR; ++mr)
#pragma unroll
            for (int mc = 0; mc < MC; ++mc) {
                const int m = pcol0 + mc * 32 + lrow;
                if (m >= a.M) continue;
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int o = orow0 + mr * 32 + 8 * g + 4 * lhi;
                    if (o >= a.O) continue;
                    float va[4], vb[4], vy[4];
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const float xs = shortcut && o + i < a.O ? to_f32<T>(x[(size_t)m * a.C + o + i]) : 0.0f;
                        va[i] = outv(1, mr, mc, 4 * g + i, 0.0f);
                        vb[i] = NTM >= 2 ? outv(2, mr, mc, 4 * g + i, 0.0f) : 0.0f;
                        vy[i] = outv(0, mr, mc, 4 * g + i, xs);
                        if (o + i < a.O) vy[i] = epi_apply(a.epi, o + i, vy[i]);
                    }
                    const size_t off = (size_t)m * a.O + o;
                    if (vec_out) {
                        if (y) store4<T>(y + off, vy[0], vy[1], vy[2], vy[3]);
                        if (ta) store4<T>(ta + off, va[0], va[1], va[2], va[3]);
                        if (tb) store4<T>(tb + off, vb[0], vb[1], vb[2], vb[3]);
                    } else {
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            if (o + i >= a.O) break;
                            if (y) y[off + i] = from_f32<T>(vy[i]);
                            if (ta) ta[off + i] = from_f32<T>(va[i]);
                            if (tb) tb[off + i] = from_f32<T>(vb[i]);
                        }
                    }
                }
            }
    } else {
#pragma unroll
        for (int t = 0; t < NTM; ++t) {
            float *__restrict__ ws = a.ws + ((size_t)split * 3 + t) * (size_t)a.M * a.O;
#pragma unroll
            for (int mr = 0; mr < MR; ++mr)
#pragma unroll
                for (int mc = 0; mc < MC; ++mc) {
                    const int m = pcol0 + mc * 32 + lrow;
                    if (m >= a.M) continue;
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        const int o = orow0 + mr * 32 + 8 * g + 4 * lhi;
                        if (o >= a.O) continue;
                        const size_t off = (size_t)m * a.O + o;
                        if (vec_out) {
                            store4<float>(ws + off, acc[t][mr][mc][4 * g], acc[t][mr][mc][4 * g + 1],
                                          acc[t][mr][mc][4 * g + 2], acc[t][mr][mc][4 * g + 3]);
                        } else {
#pragma unroll
                            for (int i = 0; i < 4; ++i)
                                if (o + i < a.O) ws[off + i] = acc[t][mr][mc][4 * g + i];
                        }
                    }
                }
        }
    }
}

// OM (qargs.h): the neuron type's terms, output-side maps and operands.
template <typename T, int BR, int BCOL, int WGR, int WGC, int BKB, bool VECK, bool S1, int OM = OM_QUADRA>
__global__ __launch_bounds__(kThreads) void qconv_bwd_data_generic_kernel(const BwdDataArgs a) {
    constexpr int VEC = Elem<T>::VEC;
    constexpr int NTM = om_terms(OM), NGM = om_gmaps(OM);
    constexpr int NB = BKB / 16;
    constexpr int KE = NB * VEC;
    constexpr int PITCH = BKB + 16;
    constexpr int ROWS = 3 * BR + 3 * BCOL;
    constexpr int RSTEP = kThreads / NB;
    constexpr int NVT = BR * NB / kThreads;
    constexpr int NVP = BCOL * NB / kThreads;
    constexpr int MR = BR / WGR / 32, MC = BCOL / WGC / 32;
    static_assert(WGR * WGC == kThreads / 64, "one wave per wave-tile");
    static_assert((BR * NB) % kThreads == 0 && (BCOL * NB) % kThreads == 0, "even load split");
    static_assert(MR >= 1 && MC >= 1 && BKB % 32 == 0, "tile shape");

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

    const T *__restrict__ gy = static_cast<const T *>(a.gy);
    const T *__restrict__ gta = static_cast<const T *>(a.ta);
    const T *__restrict__ gtb = static_cast<const T *>(a.tb);
    const T *__restrict__ w0 = static_cast<const T *>(a.wt[0]);
    const T *__restrict__ w1 = static_cast<const T *>(a.wt[1]);
    const T *__restrict__ w2 = static_cast<const T *>(a.wt[2]);

    const int c16 = tid % NB;
    const int rsub = tid / NB;

    int woff[NVT];
#pragma unroll
    for (int j = 0; j < NVT; ++j) {
        const int c = rt * BR + rsub + j * RSTEP;
        woff[j] = (c < a.C) ? c * a.K : -1;
    }
    int goff[NVP], hh[NVP], ww[NVP];
#pragma unroll
    for (int j = 0; j < NVP; ++j) {
        const int m = ct * BCOL + rsub + j * RSTEP;
        if (m < a.M) {
            const int n = (int)fdiv((uint32_t)m, a.fd_hw);
            const int rem = m - n * a.H * a.W;
            const int h = (int)fdiv((uint32_t)rem, a.fd_w);
            const int w = rem - h * a.W;
            goff[j] = n * a.HO * a.WO * a.O;
            hh[j] = h + a.PH;
            ww[j] = w + a.PW;
        } else {
            goff[j] = -1;
            hh[j] = 0;
            ww[j] = 0;
        }
    }

    // Output-gradient pixel hit by input pixel (h, w) through tap (r, q), or -1.
    auto out_pixel = [&](int j, int r, int q) -> int {
        if (goff[j] < 0) return -1;
        const int hi = hh[j] - r, wi = ww[j] - q;
        int i, jj;
        if constexpr (S1) {
            i = hi;
            jj = wi;
            if ((unsigned)i >= (unsigned)a.HO || (unsigned)jj >= (unsigned)a.WO) return -1;
        } else {
            if (hi < 0 || wi < 0) return -1;
            i = (int)fdiv((uint32_t)hi, a.fd_sh);
            jj = (int)fdiv((uint32_t)wi, a.fd_sw);
            if (i * a.SH != hi || jj * a.SW != wi || i >= a.HO || jj >= a.WO) return -1;
        }
        return goff[j] + (i * a.WO + jj) * a.O;
    };

    v4u rw[3][NVT], rg[3][NVP];  // rg: G, T_a, T_b raw
    const v4u zero = v4u{0, 0, 0, 0};

    auto load_stage = [&](int s) {
        const int k = s * KE + c16 * VEC;
        if constexpr (VECK) {
            // O % VEC == 0: the VEC elements share one tap.
            const bool kin = k < a.K;
            const int tap = (int)fdiv((uint32_t)k, a.fd_o);
            const int o = k - tap * a.O;
            const int r = (int)fdiv((uint32_t)tap, a.fd_kw);
            const int q = tap - r * a.KW;
#pragma unroll
            for (int j = 0; j < NVT; ++j) {
                const bool ok = kin && woff[j] >= 0;
                rw[0][j] = ld16(w0 + woff[j] + k, ok);
                if constexpr (NTM >= 2) rw[1][j] = ld16(w1 + woff[j] + k, ok);
                if constexpr (NTM >= 3) rw[2][j] = ld16(w2 + woff[j] + k, ok);
            }
#pragma unroll
            for (int j = 0; j < NVP; ++j) {
                const int p = kin ? out_pixel(j, r, q) : -1;
                rg[0][j] = rg[1][j] = rg[2][j] = zero;
                if (p >= 0) {
                    rg[0][j] = *reinterpret_cast<const v4u *>(gy + p + o);
                    if constexpr (NGM >= 2) rg[1][j] = *reinterpret_cast<const v4u *>(gta + p + o);
                    if constexpr (NGM >= 3) rg[2][j] = *reinterpret_cast<const v4u *>(gtb + p + o);
                }
            }
        } else {
            struct alignas(16) V { T e[VEC]; };
            V vw[3][NVT], vg[3][NVP];
#pragma unroll
            for (int e = 0; e < VEC; ++e) {
                const int ke = k + e;
                const bool kin = ke < a.K;
                const int tap = (int)fdiv((uint32_t)ke, a.fd_o);
                const int o = ke - tap * a.O;
                const int r = (int)fdiv((uint32_t)tap, a.fd_kw);
                const int q = tap - r * a.KW;
#pragma unroll
                for (int j = 0; j < NVT; ++j) {
                    const bool ok = kin && woff[j] >= 0;
                    vw[0][j].e[e] = ok ? w0[woff[j] + ke] : T(0);
                    vw[1][j].e[e] = NTM >= 2 && ok ? w1[woff[j] + ke] : T(0);
                    vw[2][j].e[e] = NTM >= 3 && ok ? w2[woff[j] + ke] : T(0);
                }
#pragma unroll
                for (int j = 0; j < NVP; ++j) {
                    const int p = kin ? out_pixel(j, r, q) : -1;
                    vg[0][j].e[e] = p >= 0 ? gy[p + o] : T(0);
                    vg[1][j].e[e] = NGM >= 2 && p >= 0 ? gta[p + o] : T(0);
                    vg[2][j].e[e] = NGM >= 3 && p >= 0 ? gtb[p + o] : T(0);
                }
            }
#pragma unroll
            for (int t = 0; t < 3; ++t) {
#pragma unroll
                for (int j = 0; j < NVT; ++j) rw[t][j] = __builtin_bit_cast(v4u, vw[t][j]);
#pragma unroll
                for (int j = 0; j < NVP; ++j) rg[t][j] = __builtin_bit_cast(v4u, vg[t][j]);
            }
        }
    };

    auto store_stage = [&](int b) {
        char *base = smem + b * ROWS * PITCH;
#pragma unroll
        for (int t = 0; t < NTM; ++t)
#pragma unroll
            for (int j = 0; j < NVT; ++j)
                lds_write16(base + (t * BR + rsub + j * RSTEP) * PITCH + c16 * 16, rw[t][j]);
        // Prologue of eq:SD (G_a = G o T_b, G_b = G o T_a, G_c = G) or the neuron type's operands.
#pragma unroll
        for (int j = 0; j < NVP; ++j) {
            v4u bt[3];
            operands_frag<T, OM>(rg[0][j], rg[1][j], rg[2][j], bt);
            const int row = 3 * BR + rsub + j * RSTEP;
#pragma unroll
            for (int t = 0; t < NTM; ++t) lds_write16(base + (row + t * BCOL) * PITCH + c16 * 16, bt[t]);
        }
    };

    // acc2: T2&4's third term (its operand is X o X), scaled by 2 X in the epilogue
    f32x16_t acc[MR][MC], acc2[OM == OM_QSQ ? MR : 1][OM == OM_QSQ ? MC : 1];
#pragma unroll
    for (int mr = 0; mr < MR; ++mr)
#pragma unroll
        for (int mc = 0; mc < MC; ++mc)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[mr][mc][v] = 0.0f;
    if constexpr (OM == OM_QSQ) {
#pragma unroll
        for (int mr = 0; mr < MR; ++mr)
#pragma unroll
            for (int mc = 0; mc < MC; ++mc)
#pragma unroll
                for (int v = 0; v < 16; ++v) acc2[mr][mc][v] = 0.0f;
    }

    const int lrow = lane & 31, lhi = lane >> 5;
    auto compute_stage = [&](int b) {
        const char *base = smem + b * ROWS * PITCH;
#pragma unroll
        for (int ch = 0; ch < BKB / 32; ++ch) {
            const int coff = ch * 32 + lhi * 16;
#pragma unroll
            for (int t = 0; t < NTM; ++t) {
                v4u bf[MC];
#pragma unroll
                for (int mc = 0; mc < MC; ++mc)
                    bf[mc] = lds_read16(base + (3 * BR + t * BCOL + wc * (BCOL / WGC) + mc * 32 + lrow) * PITCH +
                                        coff);
#pragma unroll
                for (int mr = 0; mr < MR; ++mr) {
                    const v4u af =
                        lds_read16(base + (t * BR + wr * (BR / WGR) + mr * 32 + lrow) * PITCH + coff);
#pragma unroll
                    for (int mc = 0; mc < MC; ++mc) {
                        if constexpr (OM == OM_QSQ) {
                            if (t == 2) {
                                mfma_chunk<T>(af, bf[mc], acc2[mr][mc]);
                                continue;
                            }
                        }
                        mfma_chunk<T>(af, bf[mc], acc[mr][mc]);
                    }
                }
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

    // Epilogue: rows are input channels, columns input pixels.
    const int crow0 = rt * BR + wr * (BR / WGR);
    const int pcol0 = ct * BCOL + wc * (BCOL / WGC);
    if constexpr (OM == OM_PAIR || OM == OM_SQIN) {
        if (a.splits == 1 && (OM == OM_SQIN || a.neuron == NEURON_T4I))
            neuron_dx_epilogue<T, OM, MR, MC>(acc, OM == OM_SQIN ? a.xin : a.gy, a.M, a.C, pcol0, crow0, lane);
    }
    if constexpr (OM == OM_QSQ) qsq_dx_epilogue<T, MR, MC>(acc, acc2, a.xin, a.M, a.C, pcol0, crow0, lane);
    const bool vec_out = (a.C & 3) == 0;
    T *__restrict__ dx = static_cast<T *>(a.dx);
    float *__restrict__ ws = a.ws + (size_t)split * a.M * a.C;
#pragma unroll
    for (int mr = 0; mr < MR; ++mr)
#pragma unroll
        for (int mc = 0; mc < MC; ++mc) {
            const int m = pcol0 + mc * 32 + lrow;
            if (m >= a.M) continue;
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int c = crow0 + mr * 32 + 8 * g + 4 * lhi;
                if (c >= a.C) continue;
                const size_t off = (size_t)m * a.C + c;
                const float v0 = acc[mr][mc][4 * g], v1 = acc[mr][mc][4 * g + 1];
                const float v2 = acc[mr][mc][4 * g + 2], v3 = acc[mr][mc][4 * g + 3];
                if (a.splits == 1) {
                    if (vec_out) {
                        store4<T>(dx + off, v0, v1, v2, v3);
                    } else {
                        const float vv[4] = {v0, v1, v2, v3};
#pragma unroll
                        for (int i = 0; i < 4; ++i)
                            if (c + i < a.C) dx[off + i] = from_f32<T>(vv[i]);
                    }
                } else {
                    if (vec_out) {
                        store4<float>(ws + off, v0, v1, v2, v3);
                    } else {
                        const float vv[4] = {v0, v1, v2, v3};
#pragma unroll
                        for (int i = 0; i < 4; ++i)
                            if (c + i < a.C) ws[off + i] = vv[i];
                    }
                }
            }
        }
}

// OM (qargs.h): the neuron type's maps, operands and terms; T2 stages X o X.
template <typename T, int BKP, int BO, int WGR, int WGC, int BKB, int PXG, bool VECK, int OM = OM_QUADRA>
__global__ __launch_bounds__(kThreads) void qconv_bwd_weight_generic_kernel(const BwdWeightArgs a) {
    constexpr int VEC = Elem<T>::VEC;
    constexpr int NTM = om_terms(OM), NGM = om_gmaps(OM);
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
                if constexpr (OM == OM_SQIN) rx[p] = square_frag<T>(rx[p]);
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
                    rg[1][p] = ld16(gta + off, NGM >= 2 && ok);
                    rg[2][p] = ld16(gtb + off, NGM >= 3 && ok);
                } else {
                    struct alignas(16) V { T e[VEC]; } v0, v1, v2;
#pragma unroll
                    for (int e = 0; e < VEC; ++e) {
                        const bool ok = m < a.M && obase + e < a.O;
                        v0.e[e] = ok ? gy[off + e] : T(0);
                        v1.e[e] = NGM >= 2 && ok ? gta[off + e] : T(0);
                        v2.e[e] = NGM >= 3 && ok ? gtb[off + e] : T(0);
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
                    if constexpr (om_three(OM) || OM == OM_PAIR) {
                        gv[0][p][e] = g * vget<T>(rg[2][p], e);
                        gv[1][p][e] = g * vget<T>(rg[1][p], e);
                        gv[2][p][e] = g;
                    } else if constexpr (OM == OM_SQUARE) {
                        gv[0][p][e] = 2.0f * g * vget<T>(rg[1][p], e);
                    } else {
                        gv[0][p][e] = g;
                    }
                }
#pragma unroll
            for (int t = 0; t < NTM; ++t)
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
                            d[i] = ((om_three(OM) && t == 2) || OM == OM_SQIN)  // the operand is G itself
                                       ? (vraw<T>(rg[0][2 * i], e) | (vraw<T>(rg[0][2 * i + 1], e) << 16))
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

    f32x16_t acc[NTM][MR][MC];
#pragma unroll
    for (int t = 0; t < NTM; ++t)
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
            v4u af[MR], asq[MR];  // asq: T2&4's third term sees X o X
#pragma unroll
            for (int mr = 0; mr < MR; ++mr) {
                af[mr] = lds_read16(base + (wr * (BKP / WGR) + mr * 32 + lrow) * PITCH + coff);
                if constexpr (OM == OM_QSQ) asq[mr] = square_frag<T>(af[mr]);
            }
#pragma unroll
            for (int t = 0; t < NTM; ++t)
#pragma unroll
                for (int mc = 0; mc < MC; ++mc) {
                    const v4u bf =
                        lds_read16(base + (BKP + t * BO + wc * (BO / WGC) + mc * 32 + lrow) * PITCH + coff);
#pragma unroll
                    for (int mr = 0; mr < MR; ++mr)
                        mfma_chunk<T>((OM == OM_QSQ && t == 2) ? asq[mr] : af[mr], bf, acc[t][mr][mc]);
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
    for (int t = 0; t < NTM; ++t) {
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
            for (int t = 0; t < NTM; ++t)
#pragma unroll
                for (int e = 0; e < VEC; ++e) red[(pgg * 3 + t) * BO + ov * VEC + e] = dsum[t][e];
        }
        __syncthreads();
        for (int i = tid; i < NTM * BO; i += kThreads) {
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

}  // namespace ql
