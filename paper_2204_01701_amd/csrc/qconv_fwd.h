// qconv_fwd.h -- forward of the quadratic convolution layer (arXiv 2204.01701,
// section 3.1, eq:2ndneuron3), as ONE implicit GEMM with the three per-term
// weights packed side by side:
//
//   rows    : output channels o, three row blocks per tile (W_a | W_b | W_c)
//   columns : output pixels m = (n, oh, ow)
//   K       : (r, q, c), contiguous in c for both NHWC X and OHWI W_t
//
// The im2col tile of X is staged in LDS once per K step and feeds all three
// terms.  Each lane ends up holding T_a, T_b and T_c for the same (m, o), so
// the product and sum Y = T_a o T_b + T_c (with the biases preloaded into the
// accumulators) are applied in registers and only Y (plus, when requested,
// T_a and T_b) is written to HBM.  T_c never leaves the registers.
//
// For layers with few output pixels the K range is split over workgroups;
// the raw partial sums then go to a workspace and a second kernel applies the
// biases and the product (the epilogue is not linear, so it must follow the
// full sum).
#pragma once

#include "qdevice.h"

namespace ql {

struct FwdArgs {
    const void *x;
    const void *w[3];
    const float *bias[3];
    void *y, *ta, *tb;
    float *ws;  // split-K partials [split][3][M][O]
    int N, H, W, C, O, KH, KW, SH, SW, PH, PW, HO, WO;
    int M, K;  // GEMM extents: M = N*HO*WO pixels, K = KH*KW*C
    int row_tiles, col_tiles, splits, stages_per_split, stages_total;
    FastDiv fd_howo, fd_wo, fd_c, fd_kw;
};

template <typename T, int BR, int BCOL, int WGR, int WGC, int BKB, bool VECK>
__global__ __launch_bounds__(kThreads) void qconv_fwd_kernel(const FwdArgs a) {
    constexpr int VEC = Elem<T>::VEC;
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

    v4u rw[3][NVT], rx[NVP];

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
                rw[1][j] = ld16(w1 + woff[j] + k, ok);
                rw[2][j] = ld16(w2 + woff[j] + k, ok);
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
            V vw[3][NVT], vx[NVP];
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
                    vw[1][j].e[e] = ok ? w1[woff[j] + ke] : T(0);
                    vw[2][j].e[e] = ok ? w2[woff[j] + ke] : T(0);
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
                for (int t = 0; t < 3; ++t) rw[t][j] = __builtin_bit_cast(v4u, vw[t][j]);
#pragma unroll
            for (int j = 0; j < NVP; ++j) rx[j] = __builtin_bit_cast(v4u, vx[j]);
        }
    };

    auto store_stage = [&](int b) {
        char *base = smem + b * ROWS * PITCH;
#pragma unroll
        for (int t = 0; t < 3; ++t)
#pragma unroll
            for (int j = 0; j < NVT; ++j)
                lds_write16(base + (t * BR + rsub + j * RSTEP) * PITCH + c16 * 16, rw[t][j]);
#pragma unroll
        for (int j = 0; j < NVP; ++j)
            lds_write16(base + (3 * BR + rsub + j * RSTEP) * PITCH + c16 * 16, rx[j]);
    };

    // Accumulators; the biases are preloaded when the whole K range is ours.
    f32x16_t acc[3][MR][MC];
    const int lrow = lane & 31, lhi = lane >> 5;
    const int orow0 = rt * BR + wr * (BR / WGR);
#pragma unroll
    for (int t = 0; t < 3; ++t) {
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
#pragma unroll
            for (int t = 0; t < 3; ++t)
#pragma unroll
                for (int mr = 0; mr < MR; ++mr) {
                    const v4u af = lds_read16(base + (t * BR + wr * (BR / WGR) + mr * 32 + lrow) * PITCH + coff);
#pragma unroll
                    for (int mc = 0; mc < MC; ++mc) mfma_chunk<T>(af, bf[mc], acc[t][mr][mc]);
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

    // Epilogue.
    const int pcol0 = ct * BCOL + wc * (BCOL / WGC);
    const bool vec_out = (a.O & 3) == 0;
    if (a.splits == 1) {
        T *__restrict__ y = static_cast<T *>(a.y);
        T *__restrict__ ta = static_cast<T *>(a.ta);
        T *__restrict__ tb = static_cast<T *>(a.tb);
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
                        va[i] = acc[0][mr][mc][4 * g + i];
                        vb[i] = acc[1][mr][mc][4 * g + i];
                        vy[i] = va[i] * vb[i] + acc[2][mr][mc][4 * g + i];
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
        for (int t = 0; t < 3; ++t) {
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

// Split-K epilogue: T_t = b_t + sum of the partials (in split order), then
// Y = T_a o T_b + T_c.  One thread per output element.
template <typename T>
__global__ __launch_bounds__(kThreads) void qconv_fwd_combine_kernel(const float *__restrict__ ws, int splits,
                                                                     long long MO, int O, const float *b0,
                                                                     const float *b1, const float *b2, T *y, T *ta,
                                                                     T *tb) {
    for (long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x; idx < MO;
         idx += (long long)gridDim.x * blockDim.x) {
        const int o = (int)(idx % O);
        float t3[3];
        const float *bp[3] = {b0, b1, b2};
#pragma unroll
        for (int t = 0; t < 3; ++t) {
            float s = 0.0f;
            for (int sp = 0; sp < splits; ++sp) s += ws[((size_t)sp * 3 + t) * MO + idx];
            t3[t] = (bp[t] ? bp[t][o] : 0.0f) + s;
        }
        if (y) y[idx] = from_f32<T>(t3[0] * t3[1] + t3[2]);
        if (ta) ta[idx] = from_f32<T>(t3[0]);
        if (tb) tb[idx] = from_f32<T>(t3[1]);
    }
}

}  // namespace ql
