// qconv_depthwise.h -- depthwise quadratic convolution (groups = C = O): each
// channel c has its own KH x KW filter per term (arXiv 2204.01701, section
// 4.2: the layer modules take the depth-wise setting of an ordinary
// convolution), with the neuron type's Y (qargs.h):
//
//   T_t[n,i,j,c] = b_t[c] + sum_{r,q} W_t[c,r,q] X[n, i*s-p+r, j*s-p+q, c]
//
// There is no contraction over channels, so these are direct, HBM-bound
// kernels on the vector ALU: each thread takes four channels of one pixel
// (8-byte bf16 / 16-byte fp32 loads along the contiguous NHWC channels), and
// each block stages its channel slice's filters in LDS as fp32 [term][tap][c].
// Weights are C x KH x KW (the OHWI layout with one input channel).
#pragma once

#include "qargs.h"
#include "qdevice.h"

namespace ql {

struct DwArgs {
    const void *x, *gy, *ta, *tb;   // ta: X itself for T2's input gradient
    const void *w[3];
    const float *bias[3];
    void *y, *yta, *ytb, *dx;       // forward outputs Y, T_a, T_b; input gradient
    float *dw[3], *db[3];           // weight and bias gradients (or split partials)
    float *ws_dw, *ws_db;           // partials [split][3][C][KH*KW], [split][3][C]
    int N, C, H, W, KH, KW, SH, SW, PH, PW, HO, WO;
    int M;          // pixels the pass runs over (output pixels; input pixels for the input gradient)
    int neuron, splits, px_per_split;
    FastDiv fd_howo, fd_wo, fd_hw, fd_w, fd_sh, fd_sw;
};

constexpr int kDwCB = 32;                 // channels per block
constexpr int kDwCG = kDwCB / 4;          // four-channel groups per block
constexpr int kDwPL = kThreads / kDwCG;   // pixel lanes per block

// Four consecutive channels c .. c + 3 (< C) as floats; channels past C read 0.
template <typename T, bool V4>
__device__ __forceinline__ void dw_ld4(const T *p, int cleft, float *f) {
    if constexpr (V4) {
        load4<T>(p, f);
    } else {
#pragma unroll
        for (int k = 0; k < 4; ++k) f[k] = k < cleft ? to_f32<T>(p[k]) : 0.0f;
    }
}
template <typename T, bool V4>
__device__ __forceinline__ void dw_st4(T *p, int cleft, const float *f) {
    if constexpr (V4) {
        store4<T>(p, f[0], f[1], f[2], f[3]);
    } else {
#pragma unroll
        for (int k = 0; k < 4; ++k)
            if (k < cleft) p[k] = from_f32<T>(f[k]);
    }
}

// Stage the filters of channels c0 .. c0 + kDwCB of the first NTM terms as
// fp32 [term][tap][channel] (channels past C are zero).
template <typename T, int NTM>
__device__ __forceinline__ void dw_stage_weights(const DwArgs &a, int c0, float *wl) {
    const int taps = a.KH * a.KW;
    for (int i = threadIdx.x; i < NTM * taps * kDwCB; i += kThreads) {
        const int t = i / (taps * kDwCB), rem = i - t * taps * kDwCB;
        const int tap = rem / kDwCB, cl = rem - tap * kDwCB;
        const int c = c0 + cl;
        wl[i] = c < a.C ? to_f32<T>(static_cast<const T *>(a.w[t])[(size_t)c * taps + tap]) : 0.0f;
    }
}

// ---------------------------------------------------------------------------
// Forward: one thread per (output pixel, four channels), grid-stride over pixels.
// ---------------------------------------------------------------------------
template <typename T, int OM, bool V4>
__global__ __launch_bounds__(kThreads) void qconv_dw_fwd_kernel(const DwArgs a) {
    constexpr int NTM = om_terms(OM);
    extern __shared__ float wl[];  // [NTM][taps][kDwCB]
    const int c0 = blockIdx.y * kDwCB;
    dw_stage_weights<T, NTM>(a, c0, wl);
    __syncthreads();
    const int cg = threadIdx.x % kDwCG, pl = threadIdx.x / kDwCG;
    const int c = c0 + 4 * cg, cleft = a.C - c;
    if (cleft <= 0) return;
    const int taps = a.KH * a.KW;
    const T *__restrict__ x = static_cast<const T *>(a.x);
    float bias[NTM][4];
#pragma unroll
    for (int t = 0; t < NTM; ++t)
#pragma unroll
        for (int k = 0; k < 4; ++k) bias[t][k] = (a.bias[t] && k < cleft) ? a.bias[t][c + k] : 0.0f;
    for (int m = blockIdx.x * kDwPL + pl; m < a.M; m += gridDim.x * kDwPL) {
        const int n = (int)fdiv((uint32_t)m, a.fd_howo);
        const int rem = m - n * a.HO * a.WO;
        const int oh = (int)fdiv((uint32_t)rem, a.fd_wo);
        const int ow = rem - oh * a.WO;
        float acc[NTM][4];
#pragma unroll
        for (int t = 0; t < NTM; ++t)
#pragma unroll
            for (int k = 0; k < 4; ++k) acc[t][k] = bias[t][k];
        for (int r = 0; r < a.KH; ++r) {
            const int ih = oh * a.SH - a.PH + r;
            if ((unsigned)ih >= (unsigned)a.H) continue;
            for (int q = 0; q < a.KW; ++q) {
                const int iw = ow * a.SW - a.PW + q;
                if ((unsigned)iw >= (unsigned)a.W) continue;
                float xv[4];
                dw_ld4<T, V4>(x + ((size_t)(n * a.H + ih) * a.W + iw) * a.C + c, cleft, xv);
                if constexpr (OM == OM_SQIN) {
#pragma unroll
                    for (int k = 0; k < 4; ++k) xv[k] = to_f32<T>(from_f32<T>(xv[k] * xv[k]));  // X o X in T
                }
                const int tap = r * a.KW + q;
#pragma unroll
                for (int t = 0; t < NTM; ++t) {
                    const float4 wv = *reinterpret_cast<const float4 *>(wl + (t * taps + tap) * kDwCB + 4 * cg);
                    acc[t][0] += wv.x * xv[0];
                    acc[t][1] += wv.y * xv[1];
                    acc[t][2] += wv.z * xv[2];
                    acc[t][3] += wv.w * xv[3];
                }
            }
        }
        const size_t off = (size_t)m * a.C + c;
        float yv[4];
        float xs[4] = {0.0f, 0.0f, 0.0f, 0.0f};
        if (OM == OM_PAIR && a.neuron == NEURON_T4I) dw_ld4<T, V4>(x + off, cleft, xs);  // same map: pixel m
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const float fa = acc[0][k];
            if constexpr (OM == OM_QUADRA) yv[k] = fa * acc[1][k] + acc[2][k];
            else if constexpr (OM == OM_PAIR) yv[k] = fa * acc[1][k] + xs[k];
            else if constexpr (OM == OM_SQUARE) yv[k] = fa * fa;
            else yv[k] = fa;
        }
        if (a.y) dw_st4<T, V4>(static_cast<T *>(a.y) + off, cleft, yv);
        if (a.yta) dw_st4<T, V4>(static_cast<T *>(a.yta) + off, cleft, acc[0]);
        if constexpr (NTM >= 2) {
            if (a.ytb) dw_st4<T, V4>(static_cast<T *>(a.ytb) + off, cleft, acc[1]);
        }
    }
}

// The output-side operands of the neuron type on four channels (fp32):
// QUADRA: G o T_b, G o T_a, G; PAIR: G o T_b, G o T_a; SQUARE: 2 G o T_a; SQIN: G.
template <int OM>
__device__ __forceinline__ void dw_operands(const float *g, const float *ta, const float *tb, float (*op)[4]) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        if constexpr (OM == OM_QUADRA || OM == OM_PAIR) {
            op[0][k] = g[k] * tb[k];
            op[1][k] = g[k] * ta[k];
            if constexpr (OM == OM_QUADRA) op[2][k] = g[k];
        } else if constexpr (OM == OM_SQUARE) {
            op[0][k] = 2.0f * g[k] * ta[k];
        } else {
            op[0][k] = g[k];
        }
    }
}

// ---------------------------------------------------------------------------
// Input gradient: one thread per (input pixel, four channels); the output
// pixels that tap (r, q) of input (h, w) feeds, (h + p - r) / s, are gathered.
// ---------------------------------------------------------------------------
template <typename T, int OM, bool V4>
__global__ __launch_bounds__(kThreads) void qconv_dw_bwd_data_kernel(const DwArgs a) {
    constexpr int NTM = om_terms(OM), NGM = om_gmaps(OM);
    extern __shared__ float wl[];
    const int c0 = blockIdx.y * kDwCB;
    dw_stage_weights<T, NTM>(a, c0, wl);
    __syncthreads();
    const int cg = threadIdx.x % kDwCG, pl = threadIdx.x / kDwCG;
    const int c = c0 + 4 * cg, cleft = a.C - c;
    if (cleft <= 0) return;
    const int taps = a.KH * a.KW;
    const T *__restrict__ gy = static_cast<const T *>(a.gy);
    const T *__restrict__ gta = static_cast<const T *>(a.ta);
    const T *__restrict__ gtb = static_cast<const T *>(a.tb);
    for (int m = blockIdx.x * kDwPL + pl; m < a.M; m += gridDim.x * kDwPL) {
        const int n = (int)fdiv((uint32_t)m, a.fd_hw);
        const int rem = m - n * a.H * a.W;
        const int h = (int)fdiv((uint32_t)rem, a.fd_w);
        const int w = rem - h * a.W;
        float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
        for (int r = 0; r < a.KH; ++r) {
            const int hi = h + a.PH - r;
            if (hi < 0) continue;
            const int i = (int)fdiv((uint32_t)hi, a.fd_sh);
            if (i * a.SH != hi || i >= a.HO) continue;
            for (int q = 0; q < a.KW; ++q) {
                const int wi = w + a.PW - q;
                if (wi < 0) continue;
                const int j = (int)fdiv((uint32_t)wi, a.fd_sw);
                if (j * a.SW != wi || j >= a.WO) continue;
                const size_t go = ((size_t)(n * a.HO + i) * a.WO + j) * a.C + c;
                float g[4], ta[4] = {0, 0, 0, 0}, tb[4] = {0, 0, 0, 0}, op[3][4];
                dw_ld4<T, V4>(gy + go, cleft, g);
                if constexpr (NGM >= 2) dw_ld4<T, V4>(gta + go, cleft, ta);
                if constexpr (NGM >= 3) dw_ld4<T, V4>(gtb + go, cleft, tb);
                dw_operands<OM>(g, ta, tb, op);
                const int tap = r * a.KW + q;
#pragma unroll
                for (int t = 0; t < NTM; ++t) {
                    const float4 wv = *reinterpret_cast<const float4 *>(wl + (t * taps + tap) * kDwCB + 4 * cg);
                    acc[0] += wv.x * op[t][0];
                    acc[1] += wv.y * op[t][1];
                    acc[2] += wv.z * op[t][2];
                    acc[3] += wv.w * op[t][3];
                }
            }
        }
        const size_t off = (size_t)m * a.C + c;
        if (OM == OM_SQIN || (OM == OM_PAIR && a.neuron == NEURON_T4I)) {
            float v[4];  // T2: X (in `ta`), the shortcut: G at the same pixel
            dw_ld4<T, V4>((OM == OM_SQIN ? gta : gy) + off, cleft, v);
#pragma unroll
            for (int k = 0; k < 4; ++k) acc[k] = OM == OM_SQIN ? acc[k] * (2.0f * v[k]) : acc[k] + v[k];
        }
        dw_st4<T, V4>(static_cast<T *>(a.dx) + off, cleft, acc);
    }
}

// ---------------------------------------------------------------------------
// Weight and bias gradients: each block takes a slice of kDwCB channels and
// a contiguous range of output pixels (its split); a thread accumulates, for
// its four channels, the products of the operands with X at every tap (taps
// [tap0, tap0 + TAPS) of the filter: blockIdx.z picks the group) over the
// pixels of its lane, then the block's pixel lanes are summed in a fixed order
// through LDS and written to the split's partials (or to dW, db directly).
// ---------------------------------------------------------------------------
template <typename T, int OM, bool V4, int TAPS>
__global__ __launch_bounds__(kThreads) void qconv_dw_bwd_weight_kernel(const DwArgs a) {
    constexpr int NTM = om_terms(OM), NGM = om_gmaps(OM);
    __shared__ float red[kDwPL][kDwCG][4];
    const int c0 = blockIdx.y * kDwCB;
    const int cg = threadIdx.x % kDwCG, pl = threadIdx.x / kDwCG;
    const int c = c0 + 4 * cg, cleft = a.C - c;
    const int taps = a.KH * a.KW, tap0 = blockIdx.z * TAPS;
    const int split = blockIdx.x;
    const int m_begin = split * a.px_per_split, m_end = min(a.M, m_begin + a.px_per_split);
    const T *__restrict__ x = static_cast<const T *>(a.x);
    const T *__restrict__ gy = static_cast<const T *>(a.gy);
    const T *__restrict__ gta = static_cast<const T *>(a.ta);
    const T *__restrict__ gtb = static_cast<const T *>(a.tb);
    float acc[NTM][TAPS][4], dsum[NTM][4];
#pragma unroll
    for (int t = 0; t < NTM; ++t) {
#pragma unroll
        for (int k = 0; k < 4; ++k) dsum[t][k] = 0.0f;
#pragma unroll
        for (int u = 0; u < TAPS; ++u)
#pragma unroll
            for (int k = 0; k < 4; ++k) acc[t][u][k] = 0.0f;
    }
    if (cleft > 0) {
        for (int m = m_begin + pl; m < m_end; m += kDwPL) {
            const int n = (int)fdiv((uint32_t)m, a.fd_howo);
            const int rem = m - n * a.HO * a.WO;
            const int oh = (int)fdiv((uint32_t)rem, a.fd_wo);
            const int ow = rem - oh * a.WO;
            const size_t go = (size_t)m * a.C + c;
            float g[4], ta[4] = {0, 0, 0, 0}, tb[4] = {0, 0, 0, 0}, op[3][4];
            dw_ld4<T, V4>(gy + go, cleft, g);
            if constexpr (NGM >= 2) dw_ld4<T, V4>(gta + go, cleft, ta);
            if constexpr (NGM >= 3) dw_ld4<T, V4>(gtb + go, cleft, tb);
            dw_operands<OM>(g, ta, tb, op);
#pragma unroll
            for (int t = 0; t < NTM; ++t)
#pragma unroll
                for (int k = 0; k < 4; ++k) dsum[t][k] += op[t][k];
#pragma unroll
            for (int u = 0; u < TAPS; ++u) {
                const int tap = tap0 + u;
                if (tap >= taps) break;
                const int r = tap / a.KW, q = tap - (tap / a.KW) * a.KW;
                const int ih = oh * a.SH - a.PH + r, iw = ow * a.SW - a.PW + q;
                if ((unsigned)ih >= (unsigned)a.H || (unsigned)iw >= (unsigned)a.W) continue;
                float xv[4];
                dw_ld4<T, V4>(x + ((size_t)(n * a.H + ih) * a.W + iw) * a.C + c, cleft, xv);
                if constexpr (OM == OM_SQIN) {
#pragma unroll
                    for (int k = 0; k < 4; ++k) xv[k] = to_f32<T>(from_f32<T>(xv[k] * xv[k]));
                }
#pragma unroll
                for (int t = 0; t < NTM; ++t)
#pragma unroll
                    for (int k = 0; k < 4; ++k) acc[t][u][k] += op[t][k] * xv[k];
            }
        }
    }
    // Sum over the pixel lanes in a fixed order: each value goes through LDS once.
    auto reduce_out = [&](const float *v, float *dst, size_t stride_c) {
        __syncthreads();
#pragma unroll
        for (int k = 0; k < 4; ++k) red[pl][cg][k] = v[k];
        __syncthreads();
        if (threadIdx.x < kDwCB) {
            const int g2 = threadIdx.x / 4, k = threadIdx.x % 4;
            float s = 0.0f;
            for (int l = 0; l < kDwPL; ++l) s += red[l][g2][k];
            const int cc = c0 + threadIdx.x;
            if (cc < a.C) dst[(size_t)cc * stride_c] = s;
        }
    };
#pragma unroll
    for (int t = 0; t < NTM; ++t) {
#pragma unroll
        for (int u = 0; u < TAPS; ++u) {
            const int tap = tap0 + u;
            if (tap >= taps) break;
            float *dst = a.splits == 1 ? a.dw[t] + tap : a.ws_dw + ((size_t)split * 3 + t) * a.C * taps + tap;
            reduce_out(acc[t][u], dst, taps);
        }
        if (a.db[t] && blockIdx.z == 0) {
            float *dst = a.splits == 1 ? a.db[t] : a.ws_db + ((size_t)split * 3 + t) * a.C;
            reduce_out(dsum[t], dst, 1);
        }
    }
}

// Split reduction of the depthwise weight and bias gradients, in split order.
__global__ __launch_bounds__(kThreads) void qconv_dw_reduce_kernel(const float *__restrict__ ws_dw,
                                                                   const float *__restrict__ ws_db, int splits,
                                                                   int C, int taps, int nterms, float *dw0,
                                                                   float *dw1, float *dw2, float *db0, float *db1,
                                                                   float *db2, int want_db) {
    const long long ndw = (long long)C * taps;
    const long long total = nterms * ndw + (want_db ? (long long)nterms * C : 0LL);
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (long long)gridDim.x * blockDim.x) {
        float s = 0.0f;
        if (i < nterms * ndw) {
            const int t = (int)(i / ndw);
            const long long j = i - t * ndw;
            for (int sp = 0; sp < splits; ++sp) s += ws_dw[((size_t)sp * 3 + t) * ndw + j];
            (t == 0 ? dw0 : (t == 1 ? dw1 : dw2))[j] = s;
        } else {
            const long long jj = i - nterms * ndw;
            const int t = (int)(jj / C), cc = (int)(jj % C);
            for (int sp = 0; sp < splits; ++sp) s += ws_db[((size_t)sp * 3 + t) * C + cc];
            (t == 0 ? db0 : (t == 1 ? db1 : db2))[cc] = s;
        }
    }
}

}  // namespace ql
