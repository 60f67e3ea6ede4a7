// qconv_bwd_data.h -- input gradient of the quadratic convolution layer
// (arXiv 2204.01701, section 4.3: the chain rule of eq:AD in the form of
// eq:SD).  With G = dl/dY the three per-term output gradients are
// G_a = G o T_b, G_b = G o T_a and G_c = G, and
//
//   dX[n,h,w,c] = sum_t sum_{r,q,o} G_t[n,i,j,o] W_t[o,r,q,c],  i*s - p + r = h, j*s - p + q = w
//
// computed as ONE implicit GEMM whose reduction runs over (t, r, q, o):
//
//   rows    : input channels c       (operand: W_t transposed to C x KH x KW x O)
//   columns : input pixels (n, h, w) (operand: G_t gathered at the output pixel of each tap)
//
// The G_t tiles are formed in the GEMM prologue: G, T_a and T_b are loaded
// once per K step, multiplied elementwise in fp32 while being staged into LDS,
// and never written back.  Taps that fall between output pixels (stride > 1)
// or outside the output map contribute zero.
#pragma once

#include "qdevice.h"

namespace ql {

struct BwdDataArgs {
    const void *gy, *ta, *tb;
    const void *wt[3];  // per-term weights transposed to C x KH x KW x O
    void *dx;
    float *ws;  // split-K partials [split][M][C]
    int N, H, W, C, O, KH, KW, SH, SW, PH, PW, HO, WO;
    int M, K;  // M = N*H*W input pixels, K = KH*KW*O per term
    int row_tiles, col_tiles, splits, stages_per_split, stages_total;
    FastDiv fd_hw, fd_w, fd_o, fd_kw, fd_sh, fd_sw;
};

template <typename T, int BR, int BCOL, int WGR, int WGC, int BKB, bool VECK, bool S1>
__global__ __launch_bounds__(kThreads) void qconv_bwd_data_kernel(const BwdDataArgs a) {
    constexpr int VEC = Elem<T>::VEC;
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
                rw[1][j] = ld16(w1 + woff[j] + k, ok);
                rw[2][j] = ld16(w2 + woff[j] + k, ok);
            }
#pragma unroll
            for (int j = 0; j < NVP; ++j) {
                const int p = kin ? out_pixel(j, r, q) : -1;
                if (p >= 0) {
                    rg[0][j] = *reinterpret_cast<const v4u *>(gy + p + o);
                    rg[1][j] = *reinterpret_cast<const v4u *>(gta + p + o);
                    rg[2][j] = *reinterpret_cast<const v4u *>(gtb + p + o);
                } else {
                    rg[0][j] = zero;
                    rg[1][j] = zero;
                    rg[2][j] = zero;
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
                    vw[1][j].e[e] = ok ? w1[woff[j] + ke] : T(0);
                    vw[2][j].e[e] = ok ? w2[woff[j] + ke] : T(0);
                }
#pragma unroll
                for (int j = 0; j < NVP; ++j) {
                    const int p = kin ? out_pixel(j, r, q) : -1;
                    vg[0][j].e[e] = p >= 0 ? gy[p + o] : T(0);
                    vg[1][j].e[e] = p >= 0 ? gta[p + o] : T(0);
                    vg[2][j].e[e] = p >= 0 ? gtb[p + o] : T(0);
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
        for (int t = 0; t < 3; ++t)
#pragma unroll
            for (int j = 0; j < NVT; ++j)
                lds_write16(base + (t * BR + rsub + j * RSTEP) * PITCH + c16 * 16, rw[t][j]);
        // Prologue of eq:SD: G_a = G o T_b, G_b = G o T_a, G_c = G.
#pragma unroll
        for (int j = 0; j < NVP; ++j) {
            float ga[VEC], gb[VEC];
#pragma unroll
            for (int e = 0; e < VEC; ++e) {
                const float g = vget<T>(rg[0][j], e);
                ga[e] = g * vget<T>(rg[2][j], e);
                gb[e] = g * vget<T>(rg[1][j], e);
            }
            const int row = 3 * BR + rsub + j * RSTEP;
            lds_write16(base + row * PITCH + c16 * 16, vpack<T>(ga));
            lds_write16(base + (row + BCOL) * PITCH + c16 * 16, vpack<T>(gb));
            lds_write16(base + (row + 2 * BCOL) * PITCH + c16 * 16, rg[0][j]);
        }
    };

    f32x16_t acc[MR][MC];
#pragma unroll
    for (int mr = 0; mr < MR; ++mr)
#pragma unroll
        for (int mc = 0; mc < MC; ++mc)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[mr][mc][v] = 0.0f;

    const int lrow = lane & 31, lhi = lane >> 5;
    auto compute_stage = [&](int b) {
        const char *base = smem + b * ROWS * PITCH;
#pragma unroll
        for (int ch = 0; ch < BKB / 32; ++ch) {
            const int coff = ch * 32 + lhi * 16;
#pragma unroll
            for (int t = 0; t < 3; ++t) {
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
                    for (int mc = 0; mc < MC; ++mc) mfma_chunk<T>(af, bf[mc], acc[mr][mc]);
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

// Split-K reduction of dX partials, in split order.
template <typename T>
__global__ __launch_bounds__(kThreads) void qconv_bwd_data_reduce_kernel(const float *__restrict__ ws, int splits,
                                                                         long long total, T *__restrict__ dx) {
    for (long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
         idx += (long long)gridDim.x * blockDim.x) {
        float s = 0.0f;
        for (int sp = 0; sp < splits; ++sp) s += ws[(size_t)sp * total + idx];
        dx[idx] = from_f32<T>(s);
    }
}

// Per-term weight transpose O x KH x KW x C -> C x KH x KW x O (LDS-tiled,
// 32 x 32 tiles, both sides coalesced).  grid: (ceil(C/32), ceil(O/32), 3*KH*KW).
template <typename T>
__global__ __launch_bounds__(kThreads) void qconv_weight_transpose_kernel(const T *__restrict__ w0,
                                                                          const T *__restrict__ w1,
                                                                          const T *__restrict__ w2,
                                                                          T *__restrict__ out, int O, int KHKW,
                                                                          int C) {
    __shared__ T tile[32][33];
    const int t = blockIdx.z / KHKW, tap = blockIdx.z % KHKW;
    const T *w = t == 0 ? w0 : (t == 1 ? w1 : w2);
    T *dst = out + (size_t)t * O * KHKW * C;
    const int c0 = blockIdx.x * 32, o0 = blockIdx.y * 32;
    const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 32 x 8
    for (int i = ty; i < 32; i += 8) {
        const int o = o0 + i, c = c0 + tx;
        if (o < O && c < C) tile[i][tx] = w[((size_t)o * KHKW + tap) * C + c];
    }
    __syncthreads();
    for (int i = ty; i < 32; i += 8) {
        const int c = c0 + i, o = o0 + tx;
        if (o < O && c < C) dst[((size_t)c * KHKW + tap) * O + o] = tile[tx][i];
    }
}

}  // namespace ql
