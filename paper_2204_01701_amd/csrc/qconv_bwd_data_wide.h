// qconv_bwd_data_wide.h -- input gradient of the quadratic convolution layer
// (arXiv 2204.01701, section 4.3, eq:SD), wide-tile kernel for layers with
// many input channels: bf16, stride 1, output channels a multiple of 16.
//
//   dX[n,h,w,c] = sum_t sum_{r,q,o} G_t[n, h+p-r, w+p-q, o] W_t[o,r,q,c],
//   G_a = G o T_b, G_b = G o T_a, G_c = G.
//
// The same implicit GEMM as qconv_bwd_data.h (rows: input channels, columns:
// input pixels, K = (t, r, q, o)), with a workgroup tile of BR x BCOL = 256 x
// 256 over eight waves.  Every K element of the three weight tiles and the
// three G-side tiles goes through the vector-memory address path once per
// workgroup, so the bytes moved per MFMA fall with the tile: 32768 (1/BR +
// 1/BCOL) = 256 here against 512 for a 128 x 128 tile.  To fit a three-deep
// ring of such tiles in LDS, a K step is 16 output channels of one tap (one
// MFMA k-chunk): three weight tiles of 16 rows x BR channels (natural layout,
// read with ds_read_b64_tr_b16) and three G-side tiles of BCOL pixel rows x
// 32 bytes.  A K step lies within one tap, so tap and channel offset are
// wave-uniform and each DMA address is a per-lane base plus a scalar offset;
// taps whose output pixel falls outside the map are a per-lane bit mask.
// The products G o T_b and G o T_a are formed in fp32 on the fragments.
#pragma once

#include "qargs.h"
#include "qpipe.h"

namespace ql {

// 32-byte rows (two 16-byte slots) of the G-side tiles.  Consecutive rows are
// 32 bytes apart, so rows r and r + 8 would share banks; the slot is swapped
// on every other group of 8 rows.
__device__ __forceinline__ int half_off(int row, int slot) { return row * 32 + ((slot ^ ((row >> 3) & 1)) << 4); }

template <int BR, int BCOL, int WGR, int WGC, int NS>
__global__ __launch_bounds__(64 * WGR * WGC) void qconv_bwd_data_wide_kernel(const BwdDataArgs a) {
    using T = uint16_t;
    constexpr int NT = 64 * WGR * WGC;
    constexpr int KE = 16;                // output channels per K step
    constexpr int SW = BR / 8;            // 16-byte slots per weight row
    constexpr int WT = KE * BR * 2;       // bytes of one term's weight tile
    constexpr int GT = BCOL * 32;         // bytes of one G-side tile
    constexpr int STAGE = 3 * WT + 3 * GT;
    constexpr int IPB = NT * 16;          // bytes one DMA instruction of the workgroup fills
    constexpr int NIW = WT / IPB, NIG = GT / IPB;
    constexpr int NI = 3 * NIW + 3 * NIG;
    constexpr int MR = BR / WGR / 32, MC = BCOL / WGC / 32;
    static_assert(WT % IPB == 0 && GT % IPB == 0 && NIW == 1 && NIG == 1, "one DMA instruction per tile");
    static_assert(MR >= 1 && MC >= 1, "tile shape");

    __shared__ __attribute__((aligned(1024))) char smem[NS * STAGE];

    const int tid = threadIdx.x, lane = tid & 63, wave = wave_id();
    const int wr = wave / WGC, wc = wave % WGC;
    int bid = xcd_remap(blockIdx.x, gridDim.x);
    const int tiles = a.row_tiles * a.col_tiles;
    const int split = bid / tiles;
    bid -= split * tiles;
    const int rt = bid % a.row_tiles, ct = bid / a.row_tiles;
    const int s_begin = split * a.stages_per_split;
    const int nst = min(a.stages_per_split, a.stages_total - s_begin);

    const T *__restrict__ gsrc[3] = {static_cast<const T *>(a.gy), static_cast<const T *>(a.ta),
                                     static_cast<const T *>(a.tb)};
    const T *wt[3] = {static_cast<const T *>(a.wt[0]), static_cast<const T *>(a.wt[1]),
                      static_cast<const T *>(a.wt[2])};
    const int khkw = a.KH * a.KW;

    // Weight tile fill: thread tid writes byte 16 tid of the tile, i.e. row
    // tid / SW (output channel o0 + row), physical slot tid % SW; the 8 input
    // channels it copies are those of the logical slot.  Channels past C
    // re-read the last 8 (their rows of the product are never stored).
    const int wrow = tid / SW;
    const int wslot = (tid % SW) ^ nat_swz<SW>(wrow);
    const int wc0 = min(rt * BR + 8 * wslot, a.C - 8);
    const long long wbase = (long long)wrow * khkw * a.C + wc0;
    // G-side tile fill: thread tid writes row tid / 2 (one input pixel), slot tid % 2.
    const int grow = tid >> 1;
    const int gslot = (tid & 1) ^ ((grow >> 3) & 1);
    long long go;
    uint32_t gmask = 0;
    {
        const int m = min(ct * BCOL + grow, a.M - 1);  // pixels past M: results never stored
        const int n = (int)fdiv((uint32_t)m, a.fd_hw);
        const int rem = m - n * a.H * a.W;
        const int h = (int)fdiv((uint32_t)rem, a.fd_w);
        const int w = rem - h * a.W;
        const int i0 = h + a.PH, j0 = w + a.PW;  // output pixel of tap (0, 0)
        go = ((long long)n * a.HO * a.WO + (long long)i0 * a.WO + j0) * a.O + 8 * gslot;
        for (int r = 0; r < a.KH; ++r)
            for (int q = 0; q < a.KW; ++q)
                if ((unsigned)(i0 - r) < (unsigned)a.HO && (unsigned)(j0 - q) < (unsigned)a.WO)
                    gmask |= 1u << (r * a.KW + q);
    }

    auto issue = [&](int s, int slot, bool live, int lo, int hi) {
        char *base = smem + slot * STAGE + wave * 1024;
        DmaPart part(lo, hi);
        const int k0 = min(s, a.stages_total - 1) * KE;
        const int tap = (int)fdiv((uint32_t)k0, a.fd_o);
        const int o0 = k0 - tap * a.O;
        const int r = (int)fdiv((uint32_t)tap, a.fd_kw);
        const int q = tap - r * a.KW;
        const long long sw = ((long long)o0 * khkw + tap) * a.C;
#pragma unroll
        for (int t = 0; t < 3; ++t)
            if (part.take()) dma16(wt[t] + (wbase + sw), base + t * WT);
        const long long sg = o0 - ((long long)r * a.WO + q) * a.O;
        const bool ok = live && ((gmask >> tap) & 1u);
#pragma unroll
        for (int u = 0; u < 3; ++u)
            if (part.take()) dma16(dma_src(ok, gsrc[u] + (go + sg), a.zero), base + 3 * WT + u * GT);
    };

    f32x16_t acc[MR][MC];
#pragma unroll
    for (int mr = 0; mr < MR; ++mr)
#pragma unroll
        for (int mc = 0; mc < MC; ++mc)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[mr][mc][v] = 0.0f;

    const int lrow = lane & 31, lhi = lane >> 5;
    v4u af[3][MR], gr[3][MC];  // weight fragments per term; G, T_a, T_b fragments
    auto read = [&](int slot, int, int) {
        const char *st = smem + slot * STAGE;
#pragma unroll
        for (int t = 0; t < 3; ++t)
#pragma unroll
            for (int mr = 0; mr < MR; ++mr)
                af[t][mr] = nat_frag_bf16<SW>(st + t * WT, 0, wr * (BR / WGR) + mr * 32, lane);
#pragma unroll
        for (int mc = 0; mc < MC; ++mc) {
            const int row = wc * (BCOL / WGC) + mc * 32 + lrow;
#pragma unroll
            for (int u = 0; u < 3; ++u) gr[u][mc] = lds_read16(st + 3 * WT + u * GT + half_off(row, lhi));
        }
    };
    auto mma = [&](int) {
#pragma unroll
        for (int mc = 0; mc < MC; ++mc) {
            v4u bt[3];
            prologue_frag<T>(gr[0][mc], gr[1][mc], gr[2][mc], bt[0], bt[1]);
            bt[2] = gr[0][mc];
#pragma unroll
            for (int t = 0; t < 3; ++t)
#pragma unroll
                for (int mr = 0; mr < MR; ++mr) mfma_chunk<T>(af[t][mr], bt[t], acc[mr][mc]);
        }
    };
    run_ring_single<NS, NI, 1>(nst, s_begin, issue, read, mma);

    // Epilogue: rows are input channels, columns input pixels.
    const int crow0 = rt * BR + wr * (BR / WGR);
    const int pcol0 = ct * BCOL + wc * (BCOL / WGC);
    T *__restrict__ dx = static_cast<T *>(a.dx);
#pragma unroll
    for (int mr = 0; mr < MR; ++mr)
#pragma unroll
        for (int mc = 0; mc < MC; ++mc) {
            const int m = pcol0 + mc * 32 + lrow;
            if (m >= a.M) continue;
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int c = crow0 + mr * 32 + 8 * g + 4 * lhi;
                if (c >= a.C) continue;  // C is a multiple of 8: whole groups of 4
                const size_t off = (size_t)m * a.C + c;
                const float v0 = acc[mr][mc][4 * g], v1 = acc[mr][mc][4 * g + 1];
                const float v2 = acc[mr][mc][4 * g + 2], v3 = acc[mr][mc][4 * g + 3];
                if (a.splits == 1)
                    store4<T>(dx + off, v0, v1, v2, v3);
                else
                    store4<float>(a.ws + (size_t)split * a.M * a.C + off, v0, v1, v2, v3);
            }
        }
}

}  // namespace ql
