// qconv_bwd_weight.h -- weight and bias gradients of the quadratic convolution
// layer (arXiv 2204.01701, section 4.3, eq:SD), pipelined bf16 kernel:
//
//   dW_t[o,r,q,c] = sum_{n,i,j} G_t[n,i,j,o] X[n, i*s-p+r, j*s-p+q, c]
//   db_t[o]       = sum_{n,i,j} G_t[n,i,j,o]
//   G_a = G o T_b,  G_b = G o T_a,  G_c = G
//
// ONE implicit GEMM for the three terms, reducing over the output pixels:
//   rows    : k' = (r, q, c)        (operand: im2col of X)
//   columns : (t, o), three blocks   (operand: G_t)
//   K       : output pixels m, split over workgroups
// Both operands are pixel-major in memory (NHWC), so each K step copies
// pixel rows unchanged into "natural" LDS tiles (qpipe.h) and the MFMA
// fragments are read with ds_read_b64_tr_b16, which transposes on the way
// out of LDS.  The G o T_b / G o T_a products are formed in fp32 on the
// fragments; the bias sums are accumulated from the same fp32 values.  Split-K
// partials go to a workspace reduced in split order (deterministic).
#pragma once

#include "qargs.h"
#include "qpipe.h"

namespace ql {

// The kernel body; SUM: this workgroup also accumulates the bias gradients
// (row tile 0).  Instantiated twice so that the workgroups without bias sums
// run code with no trace of them (fewer live registers in the main loop).
//
// LIN (stride 1, output map the size of the input map): each lane keeps the
// element offset of its X and G rows at the first K step of its split plus
// the (oh, ow) of its pixel, advanced by one K step (KE pixels) per issue
// with a carry, instead of splitting the pixel index into (n, oh, ow) by
// division at every step.
//
// OM (qargs.h) selects the neuron type: the output-side maps its operands
// need, the operands themselves (operands_frag), its terms' accumulators,
// and for T2 the X operand squared on its way to the MFMAs.
template <int BKP, int BO, int WGR, int WGC, int NS, int NT, bool SUM, bool LIN, int OM>
__device__ __forceinline__ void bwd_weight_body(const BwdWeightArgs &a, char *smem) {
    using T = uint16_t;                 // bf16 only: the transposed LDS read is 16-bit
    constexpr int NTM = om_terms(OM), NGM = om_gmaps(OM);
    constexpr int KE = 32;              // output pixels per K step (two MFMA k-chunks)
    constexpr int SX = BKP / 8;         // 16-byte slots per X row
    constexpr int SG = BO / 8;          // 16-byte slots per G / T_a / T_b row
    constexpr int XB = KE * BKP * 2;    // bytes of the X tile
    constexpr int GB = KE * BO * 2;     // bytes of each G-side tile
    constexpr int STAGE = XB + 3 * GB;
    constexpr int NW = NT / 64;         // waves
    constexpr int NIX = XB / (NT * 16); // DMA instructions per thread per K step
    constexpr int NIG = GB / (NT * 16);
    constexpr int NI = NIX + NGM * NIG;
    constexpr int RX = 64 / SX;         // rows one wave-instruction fills
    constexpr int RG = 64 / SG;
    constexpr int MR = BKP / WGR / 32, MC = BO / WGC / 32;
    static_assert(WGR * WGC == NW, "one wave per wave-tile");
    static_assert(XB % (NT * 16) == 0 && GB % (NT * 16) == 0 && SX <= 64 && SG <= 64, "whole DMA rounds");
    static_assert(MR >= 1 && MC >= 1, "tile shape");

    const int tid = threadIdx.x, lane = tid & 63, wave = wave_id();
    const int wr = wave / WGC, wc = wave % WGC;
    int bid = xcd_remap(blockIdx.x, gridDim.x);
    const int tiles = a.row_tiles * a.col_tiles;
    const int split = bid / tiles;
    bid -= split * tiles;
    const int rt = bid % a.row_tiles, ct = bid / a.row_tiles;
    const int s_begin = split * a.stages_per_split;
    const int nst = min(a.stages_per_split, a.stages_total - s_begin);

    const T *__restrict__ x = static_cast<const T *>(a.x);
    const T *__restrict__ gsrc[3] = {static_cast<const T *>(a.gy), static_cast<const T *>(a.ta),
                                     static_cast<const T *>(a.tb)};

    // X fill: instruction i of this wave writes rows RX * (NW i + wave) .. +RX;
    // this lane fills row RX * (NW i + wave) + lane / SX at a fixed logical slot.
    // (the swizzle needs the tile row mod 4 (mod 8 for 8-slot rows); RX * NW * i
    // is a multiple of that, so the row of instruction 0 gives it for all i)
    static_assert((RX * NW) % 8 == 0 && (RG * NW) % 8 == 0, "swizzle phase");
    const int xslot = (lane % SX) ^ nat_swz<SX>(RX * wave + lane / SX);
    const int kp = rt * BKP + 8 * xslot;  // first of the 8 k' this lane copies
    const bool kp_ok = kp < a.KP;
    int xr, xq, xc;
    {
        const int tap = (int)fdiv((uint32_t)kp, a.fd_c);
        xc = kp - tap * a.C;
        xr = (int)fdiv((uint32_t)tap, a.fd_kw);
        xq = tap - xr * a.KW;
    }
    // G fill: same scheme with rows of SG slots.
    const int gslot = (lane % SG) ^ nat_swz<SG>(RG * wave + lane / SG);
    const int og = ct * BO + 8 * gslot;
    const bool og_ok = og < a.O;

    // LIN state: per DMA instruction, the lane's pixel within a K step, its
    // element offsets at step s_begin and the (oh, ow) of the step to issue next.
    const int dh = xr - a.PH, dw = xq - a.PW;
    long long xlin[NIX], glin[NIG];
    int ohv[NIX], owv[NIX];
    if constexpr (LIN) {
#pragma unroll
        for (int i = 0; i < NIX; ++i) {
            const int m0 = s_begin * KE + RX * (NW * i + wave) + lane / SX;
            const int n = (int)fdiv((uint32_t)m0, a.fd_howo);
            const int rem = m0 - n * a.HO * a.WO;
            ohv[i] = (int)fdiv((uint32_t)rem, a.fd_wo);
            owv[i] = rem - ohv[i] * a.WO;
            xlin[i] = ((long long)m0 + (long long)dh * a.W + dw) * a.C + xc;
        }
#pragma unroll
        for (int i = 0; i < NIG; ++i)
            glin[i] = (long long)(s_begin * KE + RG * (NW * i + wave) + lane / SG) * a.O + og;
    }

    auto issue = [&](int s, int slot, bool live, int lo, int hi) {
        char *base = smem + slot * STAGE + wave * 1024;
        DmaPart part(lo, hi);
        if constexpr (LIN) {
            const int ds = s - s_begin;
            const int mleft = a.M - s * KE;  // pixels of this step that exist: lane pixel < mleft
            const long long xs = (long long)ds * KE * a.C;
#pragma unroll
            for (int i = 0; i < NIX; ++i) {
                const int p = RX * (NW * i + wave) + lane / SX;
                const bool ok = live && kp_ok && p < mleft && (unsigned)(ohv[i] + dh) < (unsigned)a.H &&
                                (unsigned)(owv[i] + dw) < (unsigned)a.W;
                if (!part.take()) continue;  // (its position advances in the part that issues it)
                dma16(dma_src(ok, x + (xlin[i] + xs), a.zero), base + i * (NT * 16));
                int ow = owv[i] + a.lin_dr;
                const int carry = ow >= a.WO ? 1 : 0;
                ow -= carry ? a.WO : 0;
                int oh = ohv[i] + a.lin_dq + carry;
                oh -= oh >= a.HO ? a.HO : 0;
                owv[i] = ow;
                ohv[i] = oh;
            }
            const long long gs = (long long)ds * KE * a.O;
#pragma unroll
            for (int i = 0; i < NIG; ++i) {
                const int p = RG * (NW * i + wave) + lane / SG;
                const bool ok = live && og_ok && p < mleft;
#pragma unroll
                for (int u = 0; u < NGM; ++u)
                    if (part.take())
                        dma16(dma_src(ok, gsrc[u] + (glin[i] + gs), a.zero), base + XB + u * GB + i * (NT * 16));
            }
            return;
        }
#pragma unroll
        for (int i = 0; i < NIX; ++i) {
            const int m = s * KE + RX * (NW * i + wave) + lane / SX;
            const int n = (int)fdiv((uint32_t)m, a.fd_howo);
            const int rem = m - n * a.HO * a.WO;
            const int oh = (int)fdiv((uint32_t)rem, a.fd_wo);
            const int ow = rem - oh * a.WO;
            const int ih = oh * a.SH - a.PH + xr, iw = ow * a.SW - a.PW + xq;
            const bool ok = live && kp_ok && m < a.M && (unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W;
            if (part.take())
                dma16(dma_src(ok, x + ((size_t)(n * a.H + ih) * a.W + iw) * a.C + xc, a.zero), base + i * (NT * 16));
        }
#pragma unroll
        for (int i = 0; i < NIG; ++i) {
            const int m = s * KE + RG * (NW * i + wave) + lane / SG;
            const bool ok = live && og_ok && m < a.M;
            const size_t off = (size_t)m * a.O + og;
#pragma unroll
            for (int u = 0; u < NGM; ++u)
                if (part.take()) dma16(dma_src(ok, gsrc[u] + off, a.zero), base + XB + u * GB + i * (NT * 16));
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
    float dsum[NTM][MC];
#pragma unroll
    for (int t = 0; t < NTM; ++t)
#pragma unroll
        for (int mc = 0; mc < MC; ++mc) dsum[t][mc] = 0.0f;
    const bool sum_db = SUM && wr == 0;

    constexpr int SETS = NT > 256 ? 1 : 2;  // fragment register sets (one when two waves share a SIMD)
    v4u af[SETS][MR], gr[SETS][3][MC];      // X and G, T_a, T_b fragments
    auto read = [&](int slot, int ch, int set) {
        const char *xt = smem + slot * STAGE;
        const char *gt = xt + XB;
#pragma unroll
        for (int mr = 0; mr < MR; ++mr) af[set][mr] = nat_frag_bf16<SX>(xt, 16 * ch, wr * (BKP / WGR) + mr * 32, lane);
#pragma unroll
        for (int mc = 0; mc < MC; ++mc)
#pragma unroll
            for (int u = 0; u < NGM; ++u)
                gr[set][u][mc] = nat_frag_bf16<SG>(gt + u * GB, 16 * ch, wc * (BO / WGC) + mc * 32, lane);
    };
    // Prologue products and bias sums in fp32, then the MFMAs.
    auto mma = [&](int set) {
        if constexpr (OM == OM_SQIN) {
#pragma unroll
            for (int mr = 0; mr < MR; ++mr) af[set][mr] = square_frag<T>(af[set][mr]);
        }
        v4u asq[MR];  // T2&4: the third term's X rows squared, once per fragment
        if constexpr (OM == OM_QSQ) {
#pragma unroll
            for (int mr = 0; mr < MR; ++mr) asq[mr] = square_frag<T>(af[set][mr]);
        }
#pragma unroll
        for (int mc = 0; mc < MC; ++mc) {
            const v4u &g = gr[set][0][mc];
            // the operands in fp32 (the bias sums use them before rounding)
            float op[3][8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float gv = vget<T>(g, e);
                if constexpr (om_three(OM) || OM == OM_PAIR) {
                    op[0][e] = gv * vget<T>(gr[set][NGM >= 3 ? 2 : 0][mc], e);
                    op[1][e] = gv * vget<T>(gr[set][NGM >= 2 ? 1 : 0][mc], e);
                    op[2][e] = gv;
                } else if constexpr (OM == OM_SQUARE) {
                    op[0][e] = 2.0f * gv * vget<T>(gr[set][NGM >= 2 ? 1 : 0][mc], e);
                } else {
                    op[0][e] = gv;
                }
            }
            if constexpr (SUM) {
                if (sum_db) {  // wave-uniform: only the waves that own the bias sums add them up
#pragma unroll
                    for (int t = 0; t < NTM; ++t) {
                        float sacc = 0.0f;
#pragma unroll
                        for (int e = 0; e < 8; ++e) sacc += op[t][e];
                        dsum[t][mc] += sacc;
                    }
                }
            }
            v4u bt[NTM];
#pragma unroll
            for (int t = 0; t < NTM; ++t) bt[t] = (om_three(OM) && t == 2) || OM == OM_SQIN ? g : vpack<T>(op[t]);
#pragma unroll
            for (int t = 0; t < NTM; ++t)
#pragma unroll
                for (int mr = 0; mr < MR; ++mr)
                    mfma_chunk<T>((OM == OM_QSQ && t == 2) ? asq[mr] : af[set][mr], bt[t], acc[t][mr][mc]);
        }
    };
    if constexpr (SETS == 2)
        run_ring<NS, NI>(nst, s_begin, issue, read, mma);
    else
        run_ring_single<NS, NI>(nst, s_begin, issue, read, mma);

    // dW epilogue: rows k', columns o; lane holds 4 consecutive k' per group.
    const int krow0 = rt * BKP + wr * (BKP / WGR);
    const int ocol0 = ct * BO + wc * (BO / WGC);
    const int lrow = lane & 31, lhi = lane >> 5;
    const bool padded = a.C_out != a.C;  // dW_t stored with C_out < C channels
    const int KPO = a.KH * a.KW * a.C_out;
    const bool vec_out = (a.KP & 3) == 0 && !padded;
    // Staged stores: each term's BO x BKP block of dW_t (o rows, k' contiguous
    // in OHWI) goes through the idle LDS ring and out in 16-byte chunks with
    // consecutive lanes on consecutive addresses.
    constexpr int PITCH = BKP * 4 + 16;  // LDS bytes per staged o row
    constexpr int MAPB = BO * PITCH;
    constexpr int RING = NS * STAGE;
    constexpr int PER = RING / MAPB >= 3 ? 3 : (RING / MAPB >= 1 ? RING / MAPB : 1);
    constexpr int CPR = BKP / 4;  // 16-byte chunks per row
    if constexpr (MAPB <= RING) {
        if (vec_out) {
#pragma unroll
            for (int t0 = 0; t0 < NTM; t0 += PER) {
                lds_barrier();  // the ring (or the previous round's tiles) is no longer read
#pragma unroll
                for (int t = t0; t < t0 + PER && t < NTM; ++t) {
                    char *tile = smem + (t - t0) * MAPB;
#pragma unroll
                    for (int mr = 0; mr < MR; ++mr)
#pragma unroll
                        for (int mc = 0; mc < MC; ++mc) {
                            const int ol = wc * (BO / WGC) + mc * 32 + lrow;
#pragma unroll
                            for (int g = 0; g < 4; ++g) {
                                const int kl = wr * (BKP / WGR) + mr * 32 + 8 * g + 4 * lhi;
                                store4<float>(reinterpret_cast<float *>(tile + ol * PITCH + kl * 4),
                                              acc[t][mr][mc][4 * g], acc[t][mr][mc][4 * g + 1],
                                              acc[t][mr][mc][4 * g + 2], acc[t][mr][mc][4 * g + 3]);
                            }
                        }
                }
                lds_barrier();
#pragma unroll
                for (int t = t0; t < t0 + PER && t < NTM; ++t) {
                    const char *tile = smem + (t - t0) * MAPB;
                    float *__restrict__ dst =
                        a.splits == 1 ? a.dw[t] : a.ws_dw + ((size_t)split * 3 + t) * (size_t)a.O * KPO;
                    for (int c = tid; c < BO * CPR; c += NT) {
                        const int row = c / CPR, cc = c % CPR;
                        const int o = ct * BO + row, k = rt * BKP + 4 * cc;
                        if (o < a.O && k < a.KP)
                            *reinterpret_cast<v4u *>(dst + (size_t)o * a.KP + k) =
                                lds_read16(tile + row * PITCH + cc * 16);
                    }
                }
            }
        }
    }
#pragma unroll
    for (int t = 0; t < NTM; ++t) {
        if (MAPB <= RING && vec_out) break;  // stored above
        float *__restrict__ dst = a.splits == 1 ? a.dw[t] : a.ws_dw + ((size_t)split * 3 + t) * (size_t)a.O * KPO;
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
                    } else if (!padded) {
#pragma unroll
                        for (int i = 0; i < 4; ++i)
                            if (k + i < a.KP) dst[off + i] = acc[t][mr][mc][4 * g + i];
                    } else {
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            const int kk = k + i;
                            const int tap = (int)fdiv((uint32_t)kk, a.fd_c);
                            const int c = kk - tap * a.C;
                            if (kk < a.KP && c < a.C_out)
                                dst[(size_t)o * KPO + tap * a.C_out + c] = acc[t][mr][mc][4 * g + i];
                        }
                    }
                }
            }
    }

    // Bias gradients: lanes l and l + 32 hold the two pixel halves of channel l % 32.
    if (SUM && sum_db) {
#pragma unroll
        for (int t = 0; t < NTM; ++t)
#pragma unroll
            for (int mc = 0; mc < MC; ++mc) {
                const float tot = dsum[t][mc] + __shfl_xor(dsum[t][mc], 32);
                const int o = ocol0 + mc * 32 + lrow;
                if (lhi == 0 && o < a.O) {
                    if (a.splits == 1)
                        a.db[t][o] = tot;
                    else
                        a.ws_db[((size_t)split * 3 + t) * a.O + o] = tot;
                }
            }
    }
}

template <int BKP, int BO, int WGR, int WGC, int NS, int NT = kThreads, int OM = OM_QUADRA>
__global__ __launch_bounds__(NT) void qconv_bwd_weight_kernel(const BwdWeightArgs a) {
    constexpr int STAGE = 32 * BKP * 2 + 3 * 32 * BO * 2;
    __shared__ __attribute__((aligned(1024))) char smem[NS * STAGE];
    // the same tile decomposition as the body: row tile 0 owns the bias sums
    int bid = xcd_remap(blockIdx.x, gridDim.x);
    const int tiles = a.row_tiles * a.col_tiles;
    bid -= (bid / tiles) * tiles;
    const bool sum = a.want_db && bid % a.row_tiles == 0;
    if (a.lin) {
        if (sum)
            bwd_weight_body<BKP, BO, WGR, WGC, NS, NT, true, true, OM>(a, smem);
        else
            bwd_weight_body<BKP, BO, WGR, WGC, NS, NT, false, true, OM>(a, smem);
    } else {
        if (sum)
            bwd_weight_body<BKP, BO, WGR, WGC, NS, NT, true, false, OM>(a, smem);
        else
            bwd_weight_body<BKP, BO, WGR, WGC, NS, NT, false, false, OM>(a, smem);
    }
}

}  // namespace ql
