// qconv_aux.h -- auxiliary kernels of the quadratic layer: the split-K
// epilogue of the forward, the split-K reductions of the gradients (all in
// split order, so results are deterministic) and the per-term weight
// transpose used by the fp32 input gradient.  Grid-stride loops over 4
// consecutive elements when the innermost extent allows 16-byte accesses.
#pragma once

#include "qdevice.h"

namespace ql {

// Forward split-K epilogue: T_t = b_t + sum over splits of the partials, then
// Y = T_a o T_b + T_c (arXiv 2204.01701, eq:2ndneuron3).  ws: [split][3][M*O].
template <typename T, bool V4>
__global__ __launch_bounds__(kThreads) void qconv_fwd_combine_kernel(const float *__restrict__ ws, int splits,
                                                                     long long MO, int O, const float *b0,
                                                                     const float *b1, const float *b2, T *y, T *ta,
                                                                     T *tb) {
    constexpr int E = V4 ? 4 : 1;
    const float *bp[3] = {b0, b1, b2};
    const long long n = MO / E;
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (long long)gridDim.x * blockDim.x) {
        const long long idx = i * E;
        const int o = (int)(idx % O);
        float t3[3][E];
#pragma unroll
        for (int t = 0; t < 3; ++t) {
#pragma unroll
            for (int e = 0; e < E; ++e) t3[t][e] = bp[t] ? bp[t][o + e] : 0.0f;
            for (int sp = 0; sp < splits; ++sp) {
                const float *src = ws + ((size_t)sp * 3 + t) * MO + idx;
                if constexpr (V4) {
                    const v4f v = *reinterpret_cast<const v4f *>(src);
#pragma unroll
                    for (int e = 0; e < 4; ++e) t3[t][e] += v[e];
                } else {
                    t3[t][0] += src[0];
                }
            }
        }
        if constexpr (V4) {
            if (y) store4<T>(y + idx, t3[0][0] * t3[1][0] + t3[2][0], t3[0][1] * t3[1][1] + t3[2][1],
                             t3[0][2] * t3[1][2] + t3[2][2], t3[0][3] * t3[1][3] + t3[2][3]);
            if (ta) store4<T>(ta + idx, t3[0][0], t3[0][1], t3[0][2], t3[0][3]);
            if (tb) store4<T>(tb + idx, t3[1][0], t3[1][1], t3[1][2], t3[1][3]);
        } else {
            if (y) y[idx] = from_f32<T>(t3[0][0] * t3[1][0] + t3[2][0]);
            if (ta) ta[idx] = from_f32<T>(t3[0][0]);
            if (tb) tb[idx] = from_f32<T>(t3[1][0]);
        }
    }
}

// Sum of `splits` partial buffers of `total` floats each, in split order; the
// result is converted to T.
template <typename T, bool V4>
__global__ __launch_bounds__(kThreads) void qconv_sum_splits_kernel(const float *__restrict__ ws, int splits,
                                                                    long long total, T *__restrict__ out) {
    constexpr int E = V4 ? 4 : 1;
    const long long n = total / E;
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (long long)gridDim.x * blockDim.x) {
        const long long idx = i * E;
        float acc[E];
#pragma unroll
        for (int e = 0; e < E; ++e) acc[e] = 0.0f;
        for (int sp = 0; sp < splits; ++sp) {
            const float *src = ws + (size_t)sp * total + idx;
            if constexpr (V4) {
                const v4f v = *reinterpret_cast<const v4f *>(src);
#pragma unroll
                for (int e = 0; e < 4; ++e) acc[e] += v[e];
            } else {
                acc[0] += src[0];
            }
        }
        if constexpr (V4) {
            store4<T>(out + idx, acc[0], acc[1], acc[2], acc[3]);
        } else {
            out[idx] = from_f32<T>(acc[0]);
        }
    }
}

// Weight/bias-gradient reduction: ws_dw [split][3][ndw], ws_db [split][3][O].
template <bool V4>
__global__ __launch_bounds__(kThreads) void qconv_bwd_weight_reduce_kernel(const float *__restrict__ ws_dw,
                                                                           const float *__restrict__ ws_db,
                                                                           int splits, long long ndw, int O,
                                                                           float *dw0, float *dw1, float *dw2,
                                                                           float *db0, float *db1, float *db2,
                                                                           int want_db) {
    constexpr int E = V4 ? 4 : 1;
    const long long nv = 3 * ndw / E;
    const long long total = nv + (want_db ? 3LL * O : 0LL);
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (long long)gridDim.x * blockDim.x) {
        if (i < nv) {
            const long long idx = i * E;
            const int t = (int)(idx / ndw);
            const long long j = idx - t * ndw;
            float acc[E];
#pragma unroll
            for (int e = 0; e < E; ++e) acc[e] = 0.0f;
            for (int sp = 0; sp < splits; ++sp) {
                const float *src = ws_dw + ((size_t)sp * 3 + t) * ndw + j;
                if constexpr (V4) {
                    const v4f v = *reinterpret_cast<const v4f *>(src);
#pragma unroll
                    for (int e = 0; e < 4; ++e) acc[e] += v[e];
                } else {
                    acc[0] += src[0];
                }
            }
            float *d = t == 0 ? dw0 : (t == 1 ? dw1 : dw2);
            if constexpr (V4)
                store4<float>(d + j, acc[0], acc[1], acc[2], acc[3]);
            else
                d[j] = acc[0];
        } else {
            const long long jj = i - nv;
            const int t = (int)(jj / O), o = (int)(jj % O);
            float s = 0.0f;
            for (int sp = 0; sp < splits; ++sp) s += ws_db[((size_t)sp * 3 + t) * O + o];
            float *d = t == 0 ? db0 : (t == 1 ? db1 : db2);
            d[o] = s;
        }
    }
}

// The same reduction for small outputs with many splits: each block takes
// 256 / SG outputs, SG threads per output sum interleaved subsets of the
// splits, and the SG partial sums are added in a fixed order through LDS.
template <int SG>
__global__ __launch_bounds__(kThreads) void qconv_bwd_weight_reduce2d_kernel(const float *__restrict__ ws_dw,
                                                                             const float *__restrict__ ws_db,
                                                                             int splits, long long ndw, int O,
                                                                             float *dw0, float *dw1, float *dw2,
                                                                             float *db0, float *db1, float *db2,
                                                                             int want_db) {
    constexpr int PER = kThreads / SG;
    __shared__ float part[SG][PER];
    const long long total = 3 * ndw + (want_db ? 3LL * O : 0LL);
    const int e = threadIdx.x % PER, sg = threadIdx.x / PER;
    for (long long base = (long long)blockIdx.x * PER; base < total; base += (long long)gridDim.x * PER) {
        const long long i = base + e;
        float s = 0.0f;
        if (i < total) {
            if (i < 3 * ndw) {
                const int t = (int)(i / ndw);
                const long long j = i - t * ndw;
                for (int sp = sg; sp < splits; sp += SG) s += ws_dw[((size_t)sp * 3 + t) * ndw + j];
            } else {
                const long long jj = i - 3 * ndw;
                const int t = (int)(jj / O), o = (int)(jj % O);
                for (int sp = sg; sp < splits; sp += SG) s += ws_db[((size_t)sp * 3 + t) * O + o];
            }
        }
        part[sg][e] = s;
        __syncthreads();
        if (sg == 0 && i < total) {
            float acc = 0.0f;
#pragma unroll
            for (int k = 0; k < SG; ++k) acc += part[k][e];
            if (i < 3 * ndw) {
                const int t = (int)(i / ndw);
                float *d = t == 0 ? dw0 : (t == 1 ? dw1 : dw2);
                d[i - t * ndw] = acc;
            } else {
                const long long jj = i - 3 * ndw;
                const int t = (int)(jj / O), o = (int)(jj % O);
                float *d = t == 0 ? db0 : (t == 1 ? db1 : db2);
                d[o] = acc;
            }
        }
        __syncthreads();
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

namespace ql {

// Copy rows of C elements into rows of Cp >= C elements, zero-filling the
// extra channels (lets 3-channel images use the 16-byte pipelined path).
// blockIdx.y selects one of the NSEG (src, dst, rows) segments: four for the
// forward (X and the three weights), one for the weight gradient (X).
struct PadSegments {
    const void *src[4];
    void *dst[4];
    long long rows[4];
};

template <typename T, int NSEG>
__global__ __launch_bounds__(kThreads) void qconv_pad_channels_kernel(PadSegments sg, int C, int Cp) {
    static_assert(NSEG >= 1 && NSEG <= 4, "segments");
    if (blockIdx.y >= NSEG) return;
    const T *__restrict__ src = static_cast<const T *>(sg.src[blockIdx.y]);
    T *__restrict__ dst = static_cast<T *>(sg.dst[blockIdx.y]);
    const long long total = sg.rows[blockIdx.y] * Cp;
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (long long)gridDim.x * blockDim.x) {
        const long long r = i / Cp;
        const int c = (int)(i - r * Cp);
        dst[i] = c < C ? src[r * C + c] : T(0);
    }
}

// Input gradient for layers with few input channels (C <= 4), on the vector
// ALUs: an MFMA tile would leave most of its rows empty.  GR = O / 8 adjacent
// lanes share one input pixel, each lane taking 8 output channels; their
// partial sums are combined with lane shuffles in a fixed order.  All taps'
// loads of G, T_a, T_b (16 bytes each) are issued before any arithmetic.  The
// weights sit in LDS as fp32, [tap][o][term][4].  Same arithmetic as the GEMM
// path: dX[n,h,w,c] = sum_{r,q,o} (G o T_b) W_a + (G o T_a) W_b + G W_c over the
// output pixels (i, j) with i*s - p + r = h, j*s - p + q = w.
template <typename T, int GR>
__global__ __launch_bounds__(kThreads) void qconv_bwd_data_smallc_kernel(
    const T *__restrict__ gy, const T *__restrict__ gta, const T *__restrict__ gtb, const T *__restrict__ w0,
    const T *__restrict__ w1, const T *__restrict__ w2, T *__restrict__ dx, int N, int H, int W, int C, int O,
    int KH, int KW, int SH, int SW, int PH, int PW, int HO, int WO) {
    constexpr int VEC = Elem<T>::VEC;
    constexpr int MAXTAP = 9;
    static_assert(GR >= 1 && GR <= 64 && (GR & (GR - 1)) == 0, "lane groups");
    extern __shared__ __attribute__((aligned(16))) float wsm[];  // [KH*KW][O][3][4]
    const int khkw = KH * KW;
    const int nslots = khkw * O * 3;
    for (int i = threadIdx.x; i < nslots * 4; i += blockDim.x) {
        const int c = i & 3, slot = i >> 2;
        const int t = slot % 3, to = slot / 3;
        const int o = to % O, tap = to / O;
        const T *w = t == 0 ? w0 : (t == 1 ? w1 : w2);
        wsm[i] = c < C ? to_f32<T>(w[((size_t)o * khkw + tap) * C + c]) : 0.0f;
    }
    __syncthreads();
    const int grp = threadIdx.x % GR;  // which 8 output channels
    const int o0 = grp * VEC;
    const long long M = (long long)N * H * W;
    const long long per_pass = (long long)gridDim.x * (blockDim.x / GR);
    for (long long m = (long long)blockIdx.x * (blockDim.x / GR) + threadIdx.x / GR; m < M;
         m += per_pass) {
        const int n = (int)(m / ((long long)H * W));
        const int rem = (int)(m - (long long)n * H * W);
        const int h = rem / W, w = rem - (rem / W) * W;
        v4u gv[MAXTAP], av[MAXTAP], bv[MAXTAP];
        bool ok[MAXTAP];
#pragma unroll
        for (int tap = 0; tap < MAXTAP; ++tap) {
            const int r = tap / KW, q = tap - (tap / KW) * KW;
            const int hi = h + PH - r, wi = w + PW - q;
            const int i = hi / SH, j = wi / SW;
            ok[tap] = tap < khkw && hi >= 0 && wi >= 0 && i * SH == hi && j * SW == wi && i < HO && j < WO;
            const size_t base = (((size_t)n * HO + (ok[tap] ? i : 0)) * WO + (ok[tap] ? j : 0)) * O + o0;
            gv[tap] = ld16(gy + base, ok[tap]);
            av[tap] = ld16(gta + base, ok[tap]);
            bv[tap] = ld16(gtb + base, ok[tap]);
        }
        float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int tap = 0; tap < MAXTAP; ++tap) {
            if (!ok[tap]) continue;
            const v4f *wt = reinterpret_cast<const v4f *>(wsm) + ((size_t)tap * O + o0) * 3;
#pragma unroll
            for (int e = 0; e < VEC; ++e) {
                const float g = vget<T>(gv[tap], e);
                const float ga = g * vget<T>(bv[tap], e);
                const float gb = g * vget<T>(av[tap], e);
                const v4f wa = wt[e * 3 + 0], wb = wt[e * 3 + 1], wc = wt[e * 3 + 2];
#pragma unroll
                for (int c = 0; c < 4; ++c) acc[c] += ga * wa[c] + gb * wb[c] + g * wc[c];
            }
        }
#pragma unroll
        for (int c = 0; c < 4; ++c)
#pragma unroll
            for (int d = 1; d < GR; d <<= 1) acc[c] += __shfl_xor(acc[c], d);
        if (grp == 0) {
#pragma unroll
            for (int c = 0; c < 4; ++c)
                if (c < C) dx[m * C + c] = from_f32<T>(acc[c]);
        }
    }
}

}  // namespace ql
