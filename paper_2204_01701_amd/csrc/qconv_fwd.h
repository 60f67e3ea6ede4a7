// qconv_fwd.h -- forward of the quadratic convolution layer (arXiv 2204.01701,
// section 3.1, eq:2ndneuron3), pipelined kernel for channel counts that are a
// multiple of the 16-byte vector.
//
// ONE implicit GEMM with the three per-term weights packed side by side:
//   rows    : output channels o, three row blocks per tile (W_a | W_b | W_c)
//   columns : output pixels m = (n, oh, ow)
//   K       : (r, q, c), contiguous in c for NHWC X and OHWI W_t
// Each K step moves 64 bytes of every tile row straight from global memory
// into a ring of NS LDS stages (qpipe.h); the im2col tile of X is staged once
// and feeds all three terms.  The biases are preloaded into the accumulators
// and the epilogue forms Y = T_a o T_b + T_c in registers, so only Y (and,
// when requested, T_a and T_b) is written to HBM.  T_c never leaves the
// registers.  With split-K the raw partial sums go to a workspace instead and
// qconv_fwd_combine_kernel applies the biases and the product.
#pragma once

#include <type_traits>

#include "qargs.h"
#include "qpipe.h"

namespace ql {

//
// OM (qargs.h) selects the neuron type: the weight rows and MFMAs of the
// terms it lacks are skipped (the tile layout keeps three term blocks), the
// pixel operand is squared on its way to the MFMAs for T2, and the epilogue
// forms the type's Y.
template <typename T, int BR, int BCOL, int WGR, int WGC, int NS, bool CA, int NT = kThreads, int OM = OM_QUADRA>
__global__ __launch_bounds__(NT) void qconv_fwd_kernel(const FwdArgs a) {
    constexpr int VEC = Elem<T>::VEC;
    constexpr int KE = 64 / (int)sizeof(T);  // reduction elements per K step
    constexpr int ROWS = 3 * BR + BCOL;
    constexpr int STAGE = ROWS * 64;
    constexpr int RPI = NT / 4;         // 64-byte tile rows one DMA instruction of the workgroup fills
    constexpr int NTM = om_terms(OM);   // first-order terms
    constexpr int NIW3 = 3 * BR / RPI;  // DMA instructions of the three weight blocks (tile layout)
    constexpr int NIW = NTM * BR / RPI; // ... of the blocks this type has (issued per thread per K step)
    constexpr int NIX = BCOL / RPI;     // ... pixel rows
    constexpr int NI = NIW + NIX;
    constexpr int MR = BR / WGR / 32, MC = BCOL / WGC / 32;
    static_assert(WGR * WGC == NT / 64, "one wave per wave-tile");
    static_assert((3 * BR) % RPI == 0 && BCOL % RPI == 0 && MR >= 1 && MC >= 1, "tile shape");
    static_assert(NTM == 3 || BR % RPI == 0, "each weight DMA instruction within one term block");

    __shared__ __attribute__((aligned(1024))) char smem[NS * STAGE];

    const int tid = threadIdx.x, lane = tid & 63, wave = wave_id();
    const int wr = wave / WGC, wc = wave % WGC;
    int bid = xcd_remap(blockIdx.x, gridDim.x);
    const int tiles = a.row_tiles * a.col_tiles;
    const int split = bid / tiles;
    bid -= split * tiles;
    const int rt = bid % a.row_tiles, ct = bid / a.row_tiles;
    // Position-major order: the taps in bounds for some position of this
    // pixel tile (a wave-uniform mask); the tile's K range is those taps only.
    uint32_t tmask = 0;
    int kst = a.stages_total;
    if (CA && a.pm) {
        const int m_hi = min(ct * BCOL + BCOL, a.M) - 1;
        for (int pos = (int)fdiv((uint32_t)(ct * BCOL), a.fd_n); pos <= (int)fdiv((uint32_t)m_hi, a.fd_n); ++pos) {
            const int oh = (int)fdiv((uint32_t)pos, a.fd_wo);
            const int h0 = oh * a.SH - a.PH, w0 = (pos - oh * a.WO) * a.SW - a.PW;
            for (int r = 0; r < a.KH; ++r)
                for (int q = 0; q < a.KW; ++q)
                    if ((unsigned)(h0 + r) < (unsigned)a.H && (unsigned)(w0 + q) < (unsigned)a.W)
                        tmask |= 1u << (r * a.KW + q);
        }
        kst = __builtin_popcount(tmask) * a.cps;
    }
    const int s_begin = split * a.stages_per_split;
    const int nst = max(0, min(a.stages_per_split, kst - s_begin));
    // NHWC row of GEMM column m
    auto prow = [&](int m) -> int {
        if (!CA || !a.pm) return m;
        const int pos = (int)fdiv((uint32_t)m, a.fd_n);
        return (m - pos * a.N) * a.HO * a.WO + pos;
    };

    const T *__restrict__ x = static_cast<const T *>(a.x);
    const T *wp[3] = {static_cast<const T *>(a.w[0]), static_cast<const T *>(a.w[1]),
                      static_cast<const T *>(a.w[2])};

    // Fill geometry: DMA instruction i of this wave writes tile rows
    // RPI i + 16 wave .. +16; this lane fills row RPI i + 16 wave + lane / 4,
    // logical 16-byte column kcol (the same for every instruction).
    const int kcol = km_fill_col(lane);
    int woff[NIW];
    int wterm[NIW];
#pragma unroll
    for (int i = 0; i < NIW; ++i) {
        const int row = RPI * i + 16 * wave + (lane >> 2);
        const int t = row / BR;
        const int o = rt * BR + (row - t * BR);
        wterm[i] = t;
        woff[i] = o < a.O ? o * a.K : -1;
    }
    int xoff[NIX], ih0[NIX], iw0[NIX];
#pragma unroll
    for (int j = 0; j < NIX; ++j) {
        const int p = RPI * (NIW3 + j) + 16 * wave + (lane >> 2) - 3 * BR;
        const int m = ct * BCOL + p;
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

    // Channel-aligned K steps (CA: C a multiple of KE, KH*KW <= 32): a K step
    // lies within one tap, so tap and channel offset are wave-uniform and each
    // DMA address is a per-lane base plus a scalar offset.  Weight rows past O
    // load the zero page (a fixed per-lane predicate: on layers with few
    // output channels most of the tile's rows, which re-reading a valid row
    // would turn into real traffic); pixels past M re-read a valid row (their
    // results are never stored).  Taps that land in the zero padding are a
    // per-lane bit mask.
    const T *wrow[NIW];
    long long xo[NIX];
    uint32_t xmask[NIX];
    bool wok[NIW];
    if constexpr (CA) {
#pragma unroll
        for (int i = 0; i < NIW; ++i) {
            const int row = RPI * i + 16 * wave + (lane >> 2);
            const int t = row / BR;
            const int o = rt * BR + (row - t * BR);
            wok[i] = o < a.O;
            wrow[i] = wp[t] + (size_t)min(o, a.O - 1) * a.K + kcol * VEC;
        }
#pragma unroll
        for (int j = 0; j < NIX; ++j) {
            const int p = RPI * (NIW3 + j) + 16 * wave + (lane >> 2) - 3 * BR;
            const int m = min(ct * BCOL + p, a.M - 1);
            int n, rem;
            if (a.pm) {
                rem = (int)fdiv((uint32_t)m, a.fd_n);
                n = m - rem * a.N;
            } else {
                n = (int)fdiv((uint32_t)m, a.fd_howo);
                rem = m - n * a.HO * a.WO;
            }
            const int oh = (int)fdiv((uint32_t)rem, a.fd_wo);
            const int ow = rem - oh * a.WO;
            const int h0 = oh * a.SH - a.PH, w0 = ow * a.SW - a.PW;
            xo[j] = (long long)n * a.H * a.W * a.C + ((long long)h0 * a.W + w0) * a.C + kcol * VEC;
            uint32_t msk = 0;
            for (int r = 0; r < a.KH; ++r)
                for (int q = 0; q < a.KW; ++q)
                    if ((unsigned)(h0 + r) < (unsigned)a.H && (unsigned)(w0 + q) < (unsigned)a.W)
                        msk |= 1u << (r * a.KW + q);
            xmask[j] = msk;
        }
    }

    auto issue = [&](int s, int slot, bool live, int lo, int hi) {
        char *base = smem + slot * STAGE + wave * 1024;
        DmaPart part(lo, hi);
        if constexpr (CA) {
            int k0, tap, c0;
            if (a.pm) {
                // step s of the tile's K range: tap = the ti-th set bit of tmask
                const int sc = max(0, min(s, kst - 1));
                const int ti = (int)fdiv((uint32_t)sc, a.fd_cps);
                uint32_t mm = tmask;
                for (int i = 0; i < ti; ++i) mm &= mm - 1;
                tap = mm ? __builtin_ctz(mm) : 0;
                c0 = (sc - ti * a.cps) * KE;
                k0 = tap * a.C + c0;
            } else {
                k0 = min(s, a.stages_total - 1) * KE;
                tap = (int)fdiv((uint32_t)k0, a.fd_c);
                c0 = k0 - tap * a.C;
            }
            const int r = (int)fdiv((uint32_t)tap, a.fd_kw);
            const int q = tap - r * a.KW;
            const long long soff = ((long long)r * a.W + q) * a.C + c0;
#pragma unroll
            for (int i = 0; i < NIW; ++i)
                if (part.take()) dma16(dma_src(wok[i], wrow[i] + k0, a.zero), base + i * (NT * 16));
#pragma unroll
            for (int j = 0; j < NIX; ++j) {
                const bool ok = live && ((xmask[j] >> tap) & 1u);
                if (part.take()) dma16(dma_src(ok, x + (xo[j] + soff), a.zero), base + (NIW3 + j) * (NT * 16));
            }
            return;
        }
        const int k = s * KE + kcol * VEC;
        const bool kin = live && k < a.K;
        const int tap = (int)fdiv((uint32_t)k, a.fd_c);
        const int c = k - tap * a.C;
        const int r = (int)fdiv((uint32_t)tap, a.fd_kw);
        const int q = tap - r * a.KW;
#pragma unroll
        for (int i = 0; i < NIW; ++i) {
            const bool ok = kin && woff[i] >= 0;
            if (part.take()) dma16(dma_src(ok, wp[wterm[i]] + woff[i] + k, a.zero), base + i * (NT * 16));
        }
#pragma unroll
        for (int j = 0; j < NIX; ++j) {
            const int ih = ih0[j] + r, iw = iw0[j] + q;
            const bool ok = kin && xoff[j] >= 0 && (unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W;
            if (part.take())
                dma16(dma_src(ok, x + xoff[j] + (ih * a.W + iw) * a.C + c, a.zero), base + (NIW3 + j) * (NT * 16));
        }
    };

    // Accumulators, biases preloaded when this workgroup owns the whole K range.
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

    // Fragment reads: row lrow of each 32-row block, logical column 2 * ch + lhi.
    const int swz = (lrow >> 2) & 3;
    const int colx0 = ((0 + lhi) ^ swz) << 4, colx1 = ((2 + lhi) ^ swz) << 4;
    constexpr int SETS = NT > 256 ? 1 : 2;  // fragment register sets (one when two waves share a SIMD)
    v4u bf[SETS][MC], af[SETS][NTM][MR];
    auto read = [&](int slot, int ch, int set) {
        const char *base = smem + slot * STAGE + lrow * 64 + (ch == 0 ? colx0 : colx1);
#pragma unroll
        for (int mc = 0; mc < MC; ++mc)
            bf[set][mc] = lds_read16(base + (3 * BR + wc * (BCOL / WGC) + mc * 32) * 64);
#pragma unroll
        for (int t = 0; t < NTM; ++t)
#pragma unroll
            for (int mr = 0; mr < MR; ++mr)
                af[set][t][mr] = lds_read16(base + (t * BR + wr * (BR / WGR) + mr * 32) * 64);
    };
    auto mma = [&](int set) {
        if constexpr (OM == OM_SQIN) {
            if (!a.xsq) {
#pragma unroll
                for (int mc = 0; mc < MC; ++mc) bf[set][mc] = square_frag<T>(bf[set][mc]);
            }
        }
        // T2&4: the third term's pixel operand is X o X, squared here once per fragment
        v4u bsq[MC];
        if constexpr (OM == OM_QSQ) {
#pragma unroll
            for (int mc = 0; mc < MC; ++mc) bsq[mc] = square_frag<T>(bf[set][mc]);
        }
#pragma unroll
        for (int t = 0; t < NTM; ++t)
#pragma unroll
            for (int mr = 0; mr < MR; ++mr)
#pragma unroll
                for (int mc = 0; mc < MC; ++mc)
                    mfma_chunk<T>(af[set][t][mr], (OM == OM_QSQ && t == 2) ? bsq[mc] : bf[set][mc], acc[t][mr][mc]);
    };
    if constexpr (SETS == 2)
        run_ring<NS, NI>(nst, s_begin, issue, read, mma);
    else  // 8 waves leave each barrier together: half the copies go out one chunk later (measured faster)
        run_ring_single<NS, NI, 2, (NI + 1) / 2>(nst, s_begin, issue, read, mma);

    // Epilogue.  Output j of a tile element: 0 the layer output Y of the
    // neuron type, 1 and 2 the saved term maps T_a and T_b.  xs: the element
    // of X the shortcut adds (T4 + identity, C == O, same pixel).
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
    const bool shortcut = OM == OM_PAIR && a.neuron == NEURON_T4I;
    // the four shortcut values of a lane's group (channels o .. o + 3 of pixel m), or zeros
    auto xs4 = [&](int m, int o, float *xv) {
        xv[0] = xv[1] = xv[2] = xv[3] = 0.0f;
        if (shortcut && m < a.M && o < a.O) load4<T>(x + (size_t)prow(m) * a.C + o, xv);
    };
    const int pcol0 = ct * BCOL + wc * (BCOL / WGC);
    const bool vec_out = (a.O & 3) == 0;
    // The single-split epilogue, compiled twice: EPI adds the fused forward
    // epilogue (EpiArgs, the statistics); without it the code is the plain one.
    auto single = [&](auto epi_c) {
        constexpr bool EPI = decltype(epi_c)::value;
            T *__restrict__ y = static_cast<T *>(a.y);
            T *__restrict__ ta = static_cast<T *>(a.ta);
            T *__restrict__ tb = static_cast<T *>(a.tb);
            // Staged stores: each output map of the tile is written into the idle
            // LDS ring as BCOL pixel rows of BR channels, then copied out in
            // 16-byte chunks, consecutive lanes on consecutive addresses (one
            // pixel's BR channels are contiguous in NHWC), instead of 4-channel
            // pieces scattered over 32 pixel rows per store instruction.
            constexpr int E = (int)sizeof(T);
            constexpr int PITCH = BR * E + 16;  // LDS bytes per staged pixel row
            constexpr int MAPB = BCOL * PITCH;
            constexpr int PER = 3 * MAPB <= NS * STAGE ? 3 : 1;  // maps staged per round
            constexpr int CPR = BR * E / 16;                       // 16-byte chunks per row
            constexpr int VE = 16 / E;                             // channels per chunk
            static_assert((CPR & (CPR - 1)) == 0 && NT % CPR == 0, "staged epilogue tile");
            static_assert(fwd_staged_fits(BR, BCOL, NS, E) == (MAPB <= NS * STAGE), "staged epilogue predicate");
            if constexpr (MAPB <= NS * STAGE) {  // (otherwise, and for O not a multiple of 16 / E: direct stores)
                if (a.O % (16 / E) == 0) {
                    T *outs[3] = {y, ta, NTM >= 2 ? tb : nullptr};
                    // Epilogue statistics: a thread copies chunks of one channel
                    // group (its chunk index mod CPR is fixed), so it sums its VE
                    // channels of y' over its pixel rows in registers.
                    const bool stats = EPI && a.stat_part != nullptr;
                    float ssum[VE], ssq[VE];
    #pragma unroll
                    for (int k = 0; k < VE; ++k) ssum[k] = ssq[k] = 0.0f;
    #pragma unroll
                    for (int r0 = 0; r0 < 3; r0 += PER) {
                        lds_barrier();  // every wave is done with the ring (or the previous round's copy)
    #pragma unroll
                        for (int j = r0; j < r0 + PER; ++j) {
                            if (!outs[j]) continue;
                            char *tile = smem + (j - r0) * MAPB;
    #pragma unroll
                            for (int mr = 0; mr < MR; ++mr)
    #pragma unroll
                                for (int mc = 0; mc < MC; ++mc) {
                                    const int p = wc * (BCOL / WGC) + mc * 32 + lrow;
    #pragma unroll
                                    for (int g = 0; g < 4; ++g) {
                                        const int ol = wr * (BR / WGR) + mr * 32 + 8 * g + 4 * lhi;
                                        float v[4], xv[4];
                                        if (j == 0) xs4(ct * BCOL + p, rt * BR + ol, xv);
    #pragma unroll
                                        for (int i = 0; i < 4; ++i) {
                                            v[i] = outv(j, mr, mc, 4 * g + i, j == 0 ? xv[i] : 0.0f);
                                            if constexpr (EPI) {
                                                const int o = rt * BR + ol + i;
                                                if (j == 0 && o < a.O) v[i] = epi_apply(a.epi, o, v[i]);
                                            }
                                        }
                                        store4<T>(reinterpret_cast<T *>(tile + p * PITCH + ol * E), v[0], v[1], v[2], v[3]);
                                    }
                                }
                        }
                        lds_barrier();
    #pragma unroll
                        for (int j = r0; j < r0 + PER; ++j) {
                            if (!outs[j]) continue;
                            const char *tile = smem + (j - r0) * MAPB;
                            for (int c = tid; c < BCOL * CPR; c += NT) {
                                const int row = c / CPR, cc = c % CPR;
                                const int m = ct * BCOL + row, o = rt * BR + cc * (16 / E);
                                if (m < a.M && o < a.O) {
                                    const v4u val = lds_read16(tile + row * PITCH + cc * 16);
                                    *reinterpret_cast<v4u *>(outs[j] + (size_t)prow(m) * a.O + o) = val;
                                    if constexpr (EPI) {
                                        if (j == 0 && stats) {
    #pragma unroll
                                            for (int k = 0; k < VE; ++k) {
                                                const float f = vget<T>(val, k);  // the stored value
                                                ssum[k] += f;
                                                ssq[k] += f * f;
                                            }
                                        }
                                    }
                                }
                            }
                        }
                    }
                    if (EPI && stats) {
                        // channel ol = cc VE + k of the tile: threads tid = cc (mod CPR), summed in tid order
                        lds_barrier();
                        float *red = reinterpret_cast<float *>(smem);
    #pragma unroll
                        for (int k = 0; k < VE; ++k) {
                            red[tid * 2 * VE + k] = ssum[k];
                            red[tid * 2 * VE + VE + k] = ssq[k];
                        }
                        lds_barrier();
                        if (tid < BR) {
                            const int cc = tid / VE, k = tid - cc * VE;
                            float s1 = 0.0f, s2 = 0.0f;
                            for (int u = cc; u < NT; u += CPR) {
                                s1 += red[u * 2 * VE + k];
                                s2 += red[u * 2 * VE + VE + k];
                            }
                            const int o = rt * BR + tid;
                            if (o < a.O) {
                                a.stat_part[(size_t)ct * 2 * a.O + o] = s1;
                                a.stat_part[(size_t)ct * 2 * a.O + a.O + o] = s2;
                            }
                        }
                    }
                    return;
                }
            }
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
                        float va[4], vb[4], vy[4], xv[4];
                        xs4(m, o, xv);
    #pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            va[i] = outv(1, mr, mc, 4 * g + i, 0.0f);
                            vb[i] = NTM >= 2 ? outv(2, mr, mc, 4 * g + i, 0.0f) : 0.0f;
                            vy[i] = outv(0, mr, mc, 4 * g + i, xv[i]);
                            if constexpr (EPI) {
                                if (o + i < a.O) vy[i] = epi_apply(a.epi, o + i, vy[i]);
                            }
                        }
                        if (NTM < 2) tb = nullptr;
                        const size_t off = (size_t)prow(m) * a.O + o;
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
    };
    if (a.splits == 1) {
        if (a.epi.scale || a.epi.shift || a.epi.relu || a.stat_part)
            single(std::true_type{});
        else
            single(std::false_type{});
    } else {
        // Split-K partials, staged like the outputs: each term's tile goes into
        // the idle ring as BCOL pixel rows of BR fp32 values and out in 16-byte
        // chunks, consecutive lanes on consecutive addresses (a wave writes four
        // whole 256-byte rows of a 64-channel tile per instruction) instead of
        // 32-byte pieces of 32 rows.
        constexpr int PITCHF = BR * 4 + 16;
        constexpr int MAPF = BCOL * PITCHF;
        constexpr int PERF = 3 * MAPF <= NS * STAGE ? 3 : (2 * MAPF <= NS * STAGE ? 2 : 1);
        constexpr int CPRF = BR / 4;  // 16-byte chunks per row
        static_assert(NT % CPRF == 0, "staged partials tile");
        if constexpr (MAPF <= NS * STAGE) {
            if (a.O % 4 == 0) {
#pragma unroll
                for (int t0 = 0; t0 < NTM; t0 += PERF) {
                    lds_barrier();  // every wave is done with the ring (or the previous round's copy)
#pragma unroll
                    for (int t = t0; t < t0 + PERF && t < NTM; ++t) {
                        char *tile = smem + (t - t0) * MAPF;
#pragma unroll
                        for (int mr = 0; mr < MR; ++mr)
#pragma unroll
                            for (int mc = 0; mc < MC; ++mc) {
                                const int pl = wc * (BCOL / WGC) + mc * 32 + lrow;
#pragma unroll
                                for (int g = 0; g < 4; ++g) {
                                    const int ol = wr * (BR / WGR) + mr * 32 + 8 * g + 4 * lhi;
                                    store4<float>(reinterpret_cast<float *>(tile + pl * PITCHF + ol * 4),
                                                  acc[t][mr][mc][4 * g], acc[t][mr][mc][4 * g + 1],
                                                  acc[t][mr][mc][4 * g + 2], acc[t][mr][mc][4 * g + 3]);
                                }
                            }
                    }
                    lds_barrier();
#pragma unroll
                    for (int t = t0; t < t0 + PERF && t < NTM; ++t) {
                        const char *tile = smem + (t - t0) * MAPF;
                        float *__restrict__ ws = a.ws + ((size_t)split * 3 + t) * (size_t)a.M * a.O;
                        for (int c = tid; c < BCOL * CPRF; c += NT) {
                            const int row = c / CPRF, cc = c % CPRF;
                            const int m = ct * BCOL + row, o = rt * BR + cc * 4;
                            if (m < a.M && o < a.O)
                                *reinterpret_cast<v4u *>(ws + (size_t)prow(m) * a.O + o) =
                                    lds_read16(tile + row * PITCHF + cc * 16);
                        }
                    }
                }
                return;
            }
        }
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
                        const size_t off = (size_t)prow(m) * a.O + o;
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

}  // namespace ql
