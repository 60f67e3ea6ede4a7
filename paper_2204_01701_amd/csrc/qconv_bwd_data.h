// qconv_bwd_data.h -- input gradient of the quadratic convolution layer
// (arXiv 2204.01701, section 4.3: the chain rule of eq:AD in the form of
// eq:SD), pipelined kernel for channel counts that are a multiple of the
// 16-byte vector.  With G = dl/dY the per-term output gradients are
// G_a = G o T_b, G_b = G o T_a, G_c = G, and
//
//   dX[n,h,w,c] = sum_t sum_{r,q,o} G_t[n,i,j,o] W_t[o,r,q,c],  i*s - p + r = h, j*s - p + q = w
//
// ONE implicit GEMM reducing over (t, r, q, o):
//   rows    : input channels c        (operand: W_t)
//   columns : input pixels (n, h, w)  (G, T_a, T_b gathered at the output pixel of each tap)
// With NATW (bf16, C a multiple of 8) each K step copies the weight rows
// W_t[o, r, q, c0 .. c0 + BR) unchanged into natural LDS tiles and reads the
// operand fragments with ds_read_b64_tr_b16; otherwise the weights come
// pre-transposed to C x KH x KW x O and are staged K-contiguous.
// Per K step the three weight tiles and the G, T_a and T_b tiles are copied
// into the LDS ring (qpipe.h).  The products G o T_b and G o T_a are formed
// in fp32 on the MFMA operand fragments right after they are read from LDS,
// so they never exist in memory.  Taps that fall between output pixels
// (stride > 1) or outside the output map load zeros.
#pragma once

#include "qargs.h"
#include "qpipe.h"

namespace ql {

//
// OM (qargs.h) selects the neuron type: only its terms' weight tiles and the
// output-side maps its operands need (G, T_a, T_b / G, T_a / G) are copied,
// the operands are formed per type (operands_frag), and the epilogue adds G
// (T4 + identity) or multiplies by 2 X (T2).  The tile layout keeps room for
// three terms and three maps.
template <typename T, int BR, int BCOL, int WGR, int WGC, int NS, bool S1, bool NATW, bool CA, int OM = OM_QUADRA>
__global__ __launch_bounds__(kThreads) void qconv_bwd_data_kernel(const BwdDataArgs a) {
    static_assert(!NATW || sizeof(T) == 2, "natural weight tiles need 16-bit elements");
    static_assert(!CA || (S1 && NATW), "channel-aligned steps are implemented for stride 1, natural weight tiles");
    constexpr int VEC = Elem<T>::VEC;
    constexpr int KE = 64 / (int)sizeof(T);
    constexpr int ROWS = 3 * BR + 3 * BCOL;
    constexpr int STAGE = ROWS * 64;
    constexpr int NTM = om_terms(OM), NGM = om_gmaps(OM);
    constexpr int NIW3 = 3 * BR / 64;   // DMA instructions of the three weight tiles (layout)
    constexpr int NIW = NTM * BR / 64;  // ... issued per thread per K step: the type's weight rows
    constexpr int NIP = BCOL / 64;      // ... rows of each of G, T_a, T_b
    constexpr int NI = NIW + NGM * NIP;
    constexpr int MR = BR / WGR / 32, MC = BCOL / WGC / 32;
    static_assert(WGR * WGC == kThreads / 64, "one wave per wave-tile");
    static_assert(BR % 64 == 0 && BCOL % 64 == 0 && MR >= 1 && MC >= 1, "tile shape");

    __shared__ __attribute__((aligned(1024))) char smem[NS * STAGE];

    const int tid = threadIdx.x, lane = tid & 63, wave = wave_id();
    const int wr = wave / WGC, wc = wave % WGC;
    const TileCoord tc = tile_coord(xcd_remap(blockIdx.x, gridDim.x), a.order, a.row_tiles, a.col_tiles, a.splits);
    const int split = tc.split, rt = tc.rt, ct = tc.ct;
    // Position-major order (CA): the taps whose output pixel lies in the map
    // for some position of this pixel tile (a wave-uniform mask); the tile's K
    // range is those taps only.
    uint32_t tmask = 0;
    int kst = a.stages_total;
    if (CA && a.pm) {
        const int m_hi = min(ct * BCOL + BCOL, a.M) - 1;
        for (int pos = (int)fdiv((uint32_t)(ct * BCOL), a.fd_n); pos <= (int)fdiv((uint32_t)m_hi, a.fd_n); ++pos) {
            const int h = (int)fdiv((uint32_t)pos, a.fd_w);
            const int i0 = h + a.PH, j0 = pos - h * a.W + a.PW;  // output pixel of tap (0, 0)
            for (int r = 0; r < a.KH; ++r)
                for (int q = 0; q < a.KW; ++q)
                    if ((unsigned)(i0 - r) < (unsigned)a.HO && (unsigned)(j0 - q) < (unsigned)a.WO)
                        tmask |= 1u << (r * a.KW + q);
        }
        kst = __builtin_popcount(tmask) * a.ops;
    }
    const int s_begin = split * a.stages_per_split;
    const int nst = max(0, min(a.stages_per_split, kst - s_begin));
    // NHWC row of GEMM column m
    auto prow = [&](int m) -> int {
        if (!CA || !a.pm) return m;
        const int pos = (int)fdiv((uint32_t)m, a.fd_n);
        return (m - pos * a.N) * a.H * a.W + pos;
    };

    const T *__restrict__ gsrc[3] = {static_cast<const T *>(a.gy), static_cast<const T *>(a.ta),
                                     static_cast<const T *>(a.tb)};
    const T *wt[3] = {static_cast<const T *>(a.wt[0]), static_cast<const T *>(a.wt[1]),
                      static_cast<const T *>(a.wt[2])};

    const int kcol = km_fill_col(lane);
    // K-contiguous (pre-transposed) weight rows: row = input channel.
    int woff[NIW];
#pragma unroll
    for (int i = 0; i < NIW; ++i) {
        const int row = 16 * (4 * i + wave) + (lane >> 2);
        const int c = rt * BR + (row - ((64 * i) / BR) * BR);
        woff[i] = c < a.C ? c * a.K : -1;
    }
    // Natural weight tiles: KE rows (K indices) of BR channels per term.
    constexpr int SW = BR / 8;          // 16-byte slots per weight row
    constexpr int WT = KE * BR * 2;     // bytes of one term's weight tile
    const int wslot = (lane % SW) ^ nat_swz<SW>(lane / SW);
    const int wc0 = rt * BR + 8 * wslot;
    const bool wc_ok = wc0 < a.C;
    const int khkw = a.KH * a.KW;
    int goff[NIP], hh[NIP], ww[NIP];
#pragma unroll
    for (int j = 0; j < NIP; ++j) {
        const int m = ct * BCOL + 16 * (4 * j + wave) + (lane >> 2);
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

    // Channel-aligned K steps (CA: O a multiple of KE, stride 1): a K step lies
    // within one tap, so tap and output-channel offset are wave-uniform and
    // each DMA address is a per-lane base plus a scalar offset.  Weight
    // columns past C load the zero page (a fixed per-lane predicate: on layers
    // with few input channels most of the tile, which re-reading valid columns
    // would turn into real traffic); pixels past M re-read valid data (their
    // results are never stored); taps whose output pixel lies outside the map
    // are a per-lane bit mask.
    const T *wrow[NATW ? NIW : 1];
    long long go[NIP];
    uint32_t gmask[NIP];
    if constexpr (CA) {
        const int wcc = min(wc0, a.C - 8);
#pragma unroll
        for (int i = 0; i < NIW; ++i) {
            const int t = (i * 4096) / WT;
            const int row = ((i * 4096) % WT + wave * 1024) / (SW * 16) + lane / SW;
            wrow[i] = wt[t] + (size_t)row * khkw * a.C + wcc;
        }
#pragma unroll
        for (int j = 0; j < NIP; ++j) {
            const int m = min(ct * BCOL + 16 * (4 * j + wave) + (lane >> 2), a.M - 1);
            int n, rem;
            if (a.pm) {
                rem = (int)fdiv((uint32_t)m, a.fd_n);
                n = m - rem * a.N;
            } else {
                n = (int)fdiv((uint32_t)m, a.fd_hw);
                rem = m - n * a.H * a.W;
            }
            const int h = (int)fdiv((uint32_t)rem, a.fd_w);
            const int w = rem - h * a.W;
            const int i0 = h + a.PH, j0 = w + a.PW;  // output pixel of tap (0, 0)
            go[j] = ((long long)n * a.HO * a.WO + (long long)i0 * a.WO + j0) * a.O + kcol * VEC;
            uint32_t msk = 0;
            for (int r = 0; r < a.KH; ++r)
                for (int q = 0; q < a.KW; ++q)
                    if ((unsigned)(i0 - r) < (unsigned)a.HO && (unsigned)(j0 - q) < (unsigned)a.WO)
                        msk |= 1u << (r * a.KW + q);
            gmask[j] = msk;
        }
    }

    auto issue = [&](int s, int slot, bool live, int lo, int hi) {
        char *base = smem + slot * STAGE + wave * 1024;
        DmaPart part(lo, hi);
        if constexpr (CA) {
            int tap, o0;
            if (a.pm) {
                // step s: output channels ((s mod ops) KE ..) of the tile's (s / ops)-th tap
                const int sc = max(0, min(s, kst - 1));  // (dead steps past the range re-read a valid one)
                const int ti = (int)fdiv((uint32_t)sc, a.fd_ops);
                o0 = (sc - ti * a.ops) * KE;
                uint32_t rest = tmask;
                for (int i = 0; i < ti; ++i) rest &= rest - 1;
                tap = rest ? __builtin_ctz(rest) : 0;
            } else {
                const int k0 = min(s, a.stages_total - 1) * KE;
                tap = (int)fdiv((uint32_t)k0, a.fd_o);
                o0 = k0 - tap * a.O;
            }
            const int r = (int)fdiv((uint32_t)tap, a.fd_kw);
            const int q = tap - r * a.KW;
            const long long sw = ((long long)o0 * khkw + tap) * a.C;
#pragma unroll
            for (int i = 0; i < NIW; ++i)
                if (part.take()) dma16(dma_src(wc_ok, wrow[i] + sw, a.zero), base + i * 4096);
            const long long sg = o0 - ((long long)r * a.WO + q) * a.O;
#pragma unroll
            for (int j = 0; j < NIP; ++j) {
                const bool ok = live && ((gmask[j] >> tap) & 1u);
#pragma unroll
                for (int u = 0; u < NGM; ++u)
                    if (part.take())
                        dma16(dma_src(ok, gsrc[u] + (go[j] + sg), a.zero), base + (NIW3 + u * NIP + j) * 4096);
            }
            return;
        }
        const int k = s * KE + kcol * VEC;
        const bool kin = live && k < a.K;
        const int tap = (int)fdiv((uint32_t)k, a.fd_o);
        const int o = k - tap * a.O;
        const int r = (int)fdiv((uint32_t)tap, a.fd_kw);
        const int q = tap - r * a.KW;
        if constexpr (NATW) {
#pragma unroll
            for (int i = 0; i < NIW; ++i) {
                const int t = (i * 4096) / WT;
                const int row = ((i * 4096) % WT + wave * 1024) / (SW * 16) + lane / SW;
                const int kr = s * KE + row;
                const int tapr = (int)fdiv((uint32_t)kr, a.fd_o);
                const int orow = kr - tapr * a.O;
                const bool ok = live && wc_ok && kr < a.K;
                if (part.take())
                    dma16(dma_src(ok, wt[t] + ((size_t)(orow * khkw + tapr) * a.C + wc0), a.zero), base + i * 4096);
            }
        } else {
#pragma unroll
            for (int i = 0; i < NIW; ++i) {
                const bool ok = kin && woff[i] >= 0;
                if (part.take()) dma16(dma_src(ok, wt[(64 * i) / BR] + woff[i] + k, a.zero), base + i * 4096);
            }
        }
#pragma unroll
        for (int j = 0; j < NIP; ++j) {
            const int hi = hh[j] - r, wi = ww[j] - q;
            bool ok;
            int p;
            if constexpr (S1) {
                ok = (unsigned)hi < (unsigned)a.HO && (unsigned)wi < (unsigned)a.WO;
                p = goff[j] + (hi * a.WO + wi) * a.O + o;
            } else {
                const int i2 = (int)fdiv((uint32_t)max(hi, 0), a.fd_sh);
                const int j2 = (int)fdiv((uint32_t)max(wi, 0), a.fd_sw);
                ok = hi >= 0 && wi >= 0 && i2 * a.SH == hi && j2 * a.SW == wi && i2 < a.HO && j2 < a.WO;
                p = goff[j] + (i2 * a.WO + j2) * a.O + o;
            }
            ok = ok && kin && goff[j] >= 0;
#pragma unroll
            for (int u = 0; u < NGM; ++u)
                if (part.take()) dma16(dma_src(ok, gsrc[u] + p, a.zero), base + (NIW3 + u * NIP + j) * 4096);
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
    const int swz = (lrow >> 2) & 3;
    const int colx0 = ((0 + lhi) ^ swz) << 4, colx1 = ((2 + lhi) ^ swz) << 4;
    v4u gr[2][3][MC], af[2][NTM][MR];  // two register sets: G, T_a, T_b and weight fragments
    auto read = [&](int slot, int ch, int set) {
        const char *base = smem + slot * STAGE + lrow * 64 + (ch == 0 ? colx0 : colx1);
#pragma unroll
        for (int mc = 0; mc < MC; ++mc) {
            const int prow = wc * (BCOL / WGC) + mc * 32;
#pragma unroll
            for (int u = 0; u < NGM; ++u) gr[set][u][mc] = lds_read16(base + (3 * BR + u * BCOL + prow) * 64);
        }
        if constexpr (NATW) {
            const char *wtile = smem + slot * STAGE;
#pragma unroll
            for (int t = 0; t < NTM; ++t)
#pragma unroll
                for (int mr = 0; mr < MR; ++mr)
                    af[set][t][mr] = nat_frag_bf16<SW>(wtile + t * WT, 16 * ch, wr * (BR / WGR) + mr * 32, lane);
        } else {
#pragma unroll
            for (int t = 0; t < NTM; ++t)
#pragma unroll
                for (int mr = 0; mr < MR; ++mr)
                    af[set][t][mr] = lds_read16(base + (t * BR + wr * (BR / WGR) + mr * 32) * 64);
        }
    };
    // The prologue products are formed on the G-side fragments, then the MFMAs.
    // Column by column, so that the products of column mc + 1 can overlap the MFMAs of column mc.
    auto mma = [&](int set) {
#pragma unroll
        for (int mc = 0; mc < MC; ++mc) {
            v4u bt[3];
            operands_frag<T, OM>(gr[set][0][mc], gr[set][NGM >= 2 ? 1 : 0][mc], gr[set][NGM >= 3 ? 2 : 0][mc], bt);
#pragma unroll
            for (int t = 0; t < NTM; ++t)
#pragma unroll
                for (int mr = 0; mr < MR; ++mr) {
                    if constexpr (OM == OM_QSQ) {
                        if (t == 2) {
                            mfma_chunk<T>(af[set][t][mr], bt[t], acc2[mr][mc]);
                            continue;
                        }
                    }
                    mfma_chunk<T>(af[set][t][mr], bt[t], acc[mr][mc]);
                }
        }
    };
    run_ring<NS, NI>(nst, s_begin, issue, read, mma);

    // Epilogue: rows are input channels, columns input pixels.
    const int crow0 = rt * BR + wr * (BR / WGR);
    const int pcol0 = ct * BCOL + wc * (BCOL / WGC);
    // The neuron type's last step (whole K range only; split partials get it
    // in the reduction): the shortcut of T4 + identity adds G at the same pixel
    // and channel (C == O, unchanged map), T2's square contributes 2 X.  (These
    // types run in image-major order: the planner sets pm for the proposed
    // neuron only.)
    if constexpr (OM == OM_PAIR || OM == OM_SQIN) {
        if (a.splits == 1 && (OM == OM_SQIN || a.neuron == NEURON_T4I))
            neuron_dx_epilogue<T, OM, MR, MC>(acc, OM == OM_SQIN ? a.xin : a.gy, a.M, a.C, pcol0, crow0, lane);
    }
    // T2&4: acc += 2 X o acc2, linear, so every split applies it to its own partial
    if constexpr (OM == OM_QSQ) qsq_dx_epilogue<T, MR, MC>(acc, acc2, a.xin, a.M, a.C, pcol0, crow0, lane);
    const bool vec_out = (a.C & 3) == 0;
    T *__restrict__ dx = static_cast<T *>(a.dx);

    // Staged stores: the BCOL x BR block (pixel rows, channels contiguous in
    // NHWC) goes through the idle LDS ring and out in 16-byte chunks with
    // consecutive lanes on consecutive addresses; OT is T for dX, float for
    // a split-K partial.
    auto staged = [&](auto tag, auto *out) -> bool {
        using OT = decltype(tag);
        constexpr int E = (int)sizeof(OT);
        constexpr int PITCH = BR * E + 16;
        constexpr int CPR = BR * E / 16;
        static_assert(BCOL * PITCH <= NS * STAGE, "staged tile fits the ring");
        if (a.C % (16 / E) != 0) return false;
        lds_barrier();  // every wave is done with the ring
#pragma unroll
        for (int mr = 0; mr < MR; ++mr)
#pragma unroll
            for (int mc = 0; mc < MC; ++mc) {
                const int pl = wc * (BCOL / WGC) + mc * 32 + lrow;
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int cl = wr * (BR / WGR) + mr * 32 + 8 * g + 4 * lhi;
                    store4<OT>(reinterpret_cast<OT *>(smem + pl * PITCH + cl * E), acc[mr][mc][4 * g],
                               acc[mr][mc][4 * g + 1], acc[mr][mc][4 * g + 2], acc[mr][mc][4 * g + 3]);
                }
            }
        lds_barrier();
        for (int c = tid; c < BCOL * CPR; c += kThreads) {
            const int row = c / CPR, cc = c % CPR;
            const int m = ct * BCOL + row, ch = rt * BR + cc * (16 / E);
            if (m < a.M && ch < a.C)
                *reinterpret_cast<v4u *>(out + (size_t)prow(m) * a.C + ch) = lds_read16(smem + row * PITCH + cc * 16);
        }
        return true;
    };
    if (a.splits == 1 ? staged(T{}, dx) : staged(float{}, a.ws + (size_t)split * a.M * a.C)) return;
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
                const size_t off = (size_t)prow(m) * a.C + c;
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
                    float *__restrict__ ws = a.ws + (size_t)split * a.M * a.C;
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

}  // namespace ql
