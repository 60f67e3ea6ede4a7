// qnet_glue.h -- the network glue around the quadratic layers of a CIFAR
// ResNet (arXiv 2204.01701, section 4.2, model construction: a batch
// normalization after each quadratic layer, a ReLU after it in deeper
// networks; residual blocks with an identity or subsampling shortcut; global
// average pooling before the classifier).  NHWC tensors of T (float, or
// uint16_t holding bf16), fp32 arithmetic, per-channel fp32 statistics.
//
// Batch normalization in training mode with gamma = 1, beta = 0: with the
// per-channel sums S = sum y and Q = sum y^2 over the M = N H W pixels (the
// quadratic layer's forward epilogue gathers them from the stored y),
//   mean = S / M,  var = Q / M - mean^2 (biased),  rstd = 1 / sqrt(var + eps),
//   z = (y - mean) rstd [+ r],  out = relu(z)
// where r is the block's shortcut: the block input itself, or (option A, at a
// stride-2 transition) the input subsampled by 2 in both directions with its
// channels placed at [C/4, C/4 + Cin) of the C output channels, zeros
// elsewhere.  The backward of out = relu(z) and of the normalization, with
// dz = dout [out > 0] and x^ = (y - mean) rstd:
//   dy = rstd (dz - sum(dz) / M - x^ sum(dz x^) / M)
// and the shortcut passes dz back to the block input.
#pragma once

#include "qdevice.h"

namespace ql {

struct NetShape {
    int n, h, w, c;
};

// Shortcut source of the residual add: none, the same shape, or option A.
enum { RES_NONE = 0, RES_SAME = 1, RES_SUB2 = 2 };

__device__ __forceinline__ void bn_params(const float *sum, const float *sumsq, int c, float inv_m, float eps,
                                          float &mean, float &rstd) {
    mean = sum[c] * inv_m;
    const float var = fmaxf(sumsq[c] * inv_m - mean * mean, 0.0f);
    rstd = 1.0f / sqrtf(var + eps);
}

// Forward: out = [relu](bn(y) + r).  A thread takes 4 channels of one pixel
// (grid-stride over the M x C/4 vectors); the block of column group 0 also
// stores mean and rstd for the backward.
template <typename T>
__global__ __launch_bounds__(kThreads) void qnet_bn_act_fwd_kernel(NetShape s, const T *__restrict__ y,
                                                                   const float *__restrict__ sum,
                                                                   const float *__restrict__ sumsq, float eps,
                                                                   int res_mode, const T *__restrict__ res,
                                                                   NetShape rs, int relu, T *__restrict__ out,
                                                                   float *__restrict__ mean_out,
                                                                   float *__restrict__ rstd_out) {
    const long long M = (long long)s.n * s.h * s.w;
    const int cv = s.c / 4;
    const long long total = M * cv;
    const float inv_m = 1.0f / (float)M;
    const int pad = res_mode == RES_SUB2 ? s.c / 4 : 0;
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (long long)gridDim.x * blockDim.x) {
        const long long m = i / cv;
        const int c0 = (int)(i - m * cv) * 4;
        float v[4], r[4] = {0.0f, 0.0f, 0.0f, 0.0f};
        load4<T>(y + m * s.c + c0, v);
        if (res_mode == RES_SAME) {
            load4<T>(res + m * s.c + c0, r);
        } else if (res_mode == RES_SUB2) {
            const int n = (int)(m / ((long long)s.h * s.w));
            const int rem = (int)(m - (long long)n * s.h * s.w);
            const int oi = rem / s.w, oj = rem - oi * s.w;
            const long long rm = ((long long)n * rs.h + 2 * oi) * rs.w + 2 * oj;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int cr = c0 + k - pad;
                r[k] = (cr >= 0 && cr < rs.c) ? to_f32<T>(res[rm * rs.c + cr]) : 0.0f;
            }
        }
        float o[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            float mu, rsd;
            bn_params(sum, sumsq, c0 + k, inv_m, eps, mu, rsd);
            const float z = (v[k] - mu) * rsd + r[k];
            o[k] = relu ? fmaxf(z, 0.0f) : z;
            if (m == 0) {
                mean_out[c0 + k] = mu;
                rstd_out[c0 + k] = rsd;
            }
        }
        store4<T>(out + m * s.c + c0, o[0], o[1], o[2], o[3]);
    }
}

// Backward, pass 1: per-channel partial sums of dz and dz x^ over the rows
// of part blockIdx.x (rows [p rpp, (p + 1) rpp)); 64 channels per block in
// y, 16 row lanes summed in lane order.  part[p][0][c] = sum dz, part[p][1][c]
// = sum dz x^ (the layout qconv_stats_reduce_kernel reduces).
template <typename T>
__global__ __launch_bounds__(kThreads) void qnet_bn_act_bwd_reduce_kernel(NetShape s, const T *__restrict__ dout,
                                                                          const T *__restrict__ out, int relu,
                                                                          const T *__restrict__ y,
                                                                          const float *__restrict__ mean,
                                                                          const float *__restrict__ rstd, int rpp,
                                                                          float *__restrict__ part) {
    __shared__ float red[2][16][65];
    const long long M = (long long)s.n * s.h * s.w;
    const int cl = threadIdx.x & 15, rl = threadIdx.x >> 4;
    const int c = blockIdx.y * 64 + 4 * cl;
    const long long r0 = (long long)blockIdx.x * rpp, r1 = min(M, r0 + rpp);
    float s1[4] = {0.0f, 0.0f, 0.0f, 0.0f}, s2[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    if (c < s.c) {
        float mu[4], rsd[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            mu[k] = mean[c + k];
            rsd[k] = rstd[c + k];
        }
        for (long long r = r0 + rl; r < r1; r += 16) {
            float g[4], o[4], v[4];
            load4<T>(dout + r * s.c + c, g);
            load4<T>(out + r * s.c + c, o);
            load4<T>(y + r * s.c + c, v);
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const float dz = (!relu || o[k] > 0.0f) ? g[k] : 0.0f;
                s1[k] += dz;
                s2[k] += dz * ((v[k] - mu[k]) * rsd[k]);
            }
        }
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        red[0][rl][4 * cl + k] = s1[k];
        red[1][rl][4 * cl + k] = s2[k];
    }
    __syncthreads();
    if (threadIdx.x < 128) {
        const int st = threadIdx.x >> 6, ch = threadIdx.x & 63;
        float t = 0.0f;
#pragma unroll
        for (int l = 0; l < 16; ++l) t += red[st][l][ch];
        const int o = blockIdx.y * 64 + ch;
        if (o < s.c) part[((size_t)blockIdx.x * 2 + st) * s.c + o] = t;
    }
}

// Backward, pass 2: dy = rstd (dz - S1 / M - x^ S2 / M).
template <typename T>
__global__ __launch_bounds__(kThreads) void qnet_bn_act_bwd_apply_kernel(NetShape s, const T *__restrict__ dout,
                                                                         const T *__restrict__ out, int relu,
                                                                         const T *__restrict__ y,
                                                                         const float *__restrict__ mean,
                                                                         const float *__restrict__ rstd,
                                                                         const float *__restrict__ s1,
                                                                         const float *__restrict__ s2,
                                                                         T *__restrict__ dy) {
    const long long M = (long long)s.n * s.h * s.w;
    const int cv = s.c / 4;
    const long long total = M * cv;
    const float inv_m = 1.0f / (float)M;
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (long long)gridDim.x * blockDim.x) {
        const long long m = i / cv;
        const int c0 = (int)(i - m * cv) * 4;
        float g[4], o[4], v[4], d[4];
        load4<T>(dout + m * s.c + c0, g);
        load4<T>(out + m * s.c + c0, o);
        load4<T>(y + m * s.c + c0, v);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int c = c0 + k;
            const float dz = (!relu || o[k] > 0.0f) ? g[k] : 0.0f;
            const float xh = (v[k] - mean[c]) * rstd[c];
            d[k] = rstd[c] * (dz - s1[c] * inv_m - xh * (s2[c] * inv_m));
        }
        store4<T>(dy + m * s.c + c0, d[0], d[1], d[2], d[3]);
    }
}

// The shortcut's gradient added to the block input's: dx (the input gradient
// of the block's first layer, xs) += the shortcut's share of dz = dout [out > 0]
// (s: the block output).  RES_SAME: dz itself; RES_SUB2: at even (h, w),
// dz of output pixel (h / 2, w / 2), channel c + C / 4.  One thread per
// 4 channels of an input pixel.
template <typename T>
__global__ __launch_bounds__(kThreads) void qnet_residual_bwd_kernel(NetShape s, const T *__restrict__ dout,
                                                                     const T *__restrict__ out, NetShape xs,
                                                                     int mode, T *__restrict__ dx) {
    const long long Mx = (long long)xs.n * xs.h * xs.w;
    const int cv = xs.c / 4;
    const long long total = Mx * cv;
    const int pad = mode == RES_SUB2 ? s.c / 4 : 0;
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (long long)gridDim.x * blockDim.x) {
        const long long m = i / cv;
        const int c0 = (int)(i - m * cv) * 4;
        float v[4], add[4] = {0.0f, 0.0f, 0.0f, 0.0f};
        load4<T>(dx + m * xs.c + c0, v);
        long long om = -1;
        if (mode == RES_SAME) {
            om = m;
        } else {
            const int n = (int)(m / ((long long)xs.h * xs.w));
            const int rem = (int)(m - (long long)n * xs.h * xs.w);
            const int h = rem / xs.w, w = rem - h * xs.w;
            if ((h & 1) == 0 && (w & 1) == 0 && h / 2 < s.h && w / 2 < s.w)
                om = ((long long)n * s.h + h / 2) * s.w + w / 2;
        }
        if (om >= 0) {
            float g[4], o[4];
            load4<T>(dout + om * s.c + c0 + pad, g);
            load4<T>(out + om * s.c + c0 + pad, o);
#pragma unroll
            for (int k = 0; k < 4; ++k) add[k] = o[k] > 0.0f ? g[k] : 0.0f;
        }
        store4<T>(dx + m * xs.c + c0, v[0] + add[0], v[1] + add[1], v[2] + add[2], v[3] + add[3]);
    }
}

// Global average pooling: y[n, c] = mean over the H W pixels of x[n, :, :, c];
// one thread per (n, c), pixels in order.
template <typename T>
__global__ __launch_bounds__(kThreads) void qnet_gap_fwd_kernel(NetShape s, const T *__restrict__ x,
                                                                T *__restrict__ y) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= s.n * s.c) return;
    const int n = i / s.c, c = i - n * s.c;
    const int hw = s.h * s.w;
    float acc = 0.0f;
    for (int p = 0; p < hw; ++p) acc += to_f32<T>(x[((long long)n * hw + p) * s.c + c]);
    y[i] = from_f32<T>(acc / (float)hw);
}

// Its backward: dx[n, p, c] = dy[n, c] / (H W).
template <typename T>
__global__ __launch_bounds__(kThreads) void qnet_gap_bwd_kernel(NetShape s, const T *__restrict__ dy,
                                                                T *__restrict__ dx) {
    const long long total = (long long)s.n * s.h * s.w * s.c;
    const float inv = 1.0f / (float)(s.h * s.w);
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (long long)gridDim.x * blockDim.x) {
        const long long n = i / ((long long)s.h * s.w * s.c);
        const int c = (int)(i % s.c);
        dx[i] = from_f32<T>(to_f32<T>(dy[n * s.c + c]) * inv);
    }
}

}  // namespace ql
