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
