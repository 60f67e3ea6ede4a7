// qconv_depthwise.h -- depthwise quadratic convolution (groups = C = O): each
// channel c has its own KH x KW filter per term (arXiv 2204.01701, section
// 4.2: the layer modules take the depth-wise setting of an ordinary
// convolution), with the neuron type's Y (qargs.h):
//
//   T_t[n,i,j,c] = b_t[c] + sum_{r,q} W_t[c,r,q] X[n, i*s-p+r, j*s-p+q, c]
//
// There is no contraction over channels, so these are direct, HBM-bound
// kernels on the vector ALU.  A thread takes V channels of one pixel (16-byte
// loads along the contiguous NHWC channels where C allows), a block a channel
// slice of up to 8 lanes x V channels (128 bytes of each pixel) and a chunk of
// pixels, and stages the slice's filters in LDS as fp32 [term][tap][c].
// Weights are C x KH x KW (the OHWI layout with one input channel).
//
// The 3 x 3 kernels (the MobileNet shape) issue the loads of every tap before
// any arithmetic, with out-of-range taps clamped to a valid address and their
// values selected to zero, so that a wave keeps all of them in flight; the
// generic kernels (any filter size) loop over the taps.
#pragma once

#include <type_traits>

#include "qargs.h"
#include "qdevice.h"

namespace ql {

struct DwArgs {
    const void *x, *gy, *ta, *tb;   // ta: X itself for T2's input gradient
    const void *w[3];
    const float *bias[3];
    void *y, *yta, *ytb, *dx;       // forward outputs Y, T_a, T_b; input gradient
    float *dw[3], *db[3];           // weight and bias gradients
    float *ws;                      // split partials [split][J]: dW_t[c][tap] at (t C + c) taps + tap, db_t[c] after
    int N, C, H, W, KH, KW, SH, SW, PH, PW, HO, WO;
    int M;          // pixels the pass runs over (output pixels; input pixels for the input gradient)
    int neuron, splits, px_per_split;
    int J;          // partials per split: nterms C (taps + 1)
    int lanes, lsh; // 3 x 3 kernels: channel lanes per pixel (1, 2, 4 or 8) and its log2
    int tiles;      // 3 x 3 kernels: channel slices of lanes x V channels
    // column kernels: M counts columns (image, row group of R rows, column);
    // ng row groups per image, iwid columns per row
    int ng, iwid;
    const void *zero;  // 16 zero bytes: the source of out-of-range taps (generic kernels)
    int xbytes, pbytes;  // 3 x 3 kernels: bytes of X (and dX) and of an output-side map (< 2^31)
    EpiArgs epi;         // forward epilogue of Y (qargs.h)
    FastDiv fd_howo, fd_wo, fd_hw, fd_w, fd_sh, fd_sw, fd_item, fd_iw;
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
            if (k < cleft) yv[k] = epi_apply(a.epi, c + k, yv[k]);
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
            float *dst = a.splits == 1 ? a.dw[t] + tap : a.ws + (size_t)split * a.J + (size_t)t * a.C * taps + tap;
            reduce_out(acc[t][u], dst, taps);
        }
        if (a.db[t] && blockIdx.z == 0) {
            float *dst = a.splits == 1 ? a.db[t] : a.ws + (size_t)split * a.J + (size_t)(NTM * taps + t) * a.C;
            reduce_out(dsum[t], dst, 1);
        }
    }
}

// Split reduction of the depthwise weight and bias gradients: a block takes
// 16 partial indices j, 16 lanes of it sum every 16th split, and the 16 lane
// sums are added in lane order (a fixed order: the result does not depend on
// scheduling).  j < nterms C taps are dW values, the next nterms C the db.
template <int = 0>  // (a template: defined once across the translation units that include this header)
__global__ __launch_bounds__(kThreads) void qconv_dw_reduce_kernel(const float *__restrict__ ws, int splits, int J,
                                                                   int C, int taps, int nterms, float *dw0,
                                                                   float *dw1, float *dw2, float *db0, float *db1,
                                                                   float *db2, int want_db) {
    __shared__ float part[16][17];
    const int jl = threadIdx.x & 15, sl = threadIdx.x >> 4;
    const int j = blockIdx.x * 16 + jl;
    const int ndw = nterms * C * taps;
    const int jn = ndw + (want_db ? nterms * C : 0);
    float s = 0.0f;
    if (j < jn) {
#pragma unroll 4
        for (int sp = sl; sp < splits; sp += 16) s += ws[(size_t)sp * J + j];
    }
    part[sl][jl] = s;
    __syncthreads();
    if (sl == 0 && j < jn) {
        float t = 0.0f;
#pragma unroll
        for (int l = 0; l < 16; ++l) t += part[l][jl];
        if (j < ndw) {
            const int term = j / (C * taps), rem = j - term * C * taps;
            (term == 0 ? dw0 : (term == 1 ? dw1 : dw2))[rem] = t;
        } else {
            const int term = (j - ndw) / C, cc = (j - ndw) - term * C;
            (term == 0 ? db0 : (term == 1 ? db1 : db2))[cc] = t;
        }
    }
}

// ===========================================================================
// 3 x 3 kernels.
// ===========================================================================

// V channels c .. c + V - 1 as floats.  VEC: one aligned V * sizeof(T)-byte
// load (16 or 8 bytes; C % V == 0); else element loads, channels past C read 0.
template <typename T, int V, bool VEC>
__device__ __forceinline__ void dw_ldv(const T *p, int cleft, float *f) {
    if constexpr (VEC && V * sizeof(T) == 16) {
        const v4u v = *reinterpret_cast<const v4u *>(p);
#pragma unroll
        for (int k = 0; k < V; ++k) f[k] = vget<T>(v, k);
    } else if constexpr (VEC) {
        static_assert(V == 4, "8-byte vectors hold four channels");
        load4<T>(p, f);
    } else {
#pragma unroll
        for (int k = 0; k < V; ++k) f[k] = k < cleft ? to_f32<T>(p[k]) : 0.0f;
    }
}
template <typename T, int V, bool VEC>
__device__ __forceinline__ void dw_stv(T *p, int cleft, const float *f) {
    if constexpr (VEC && V * sizeof(T) == 16) {
        *reinterpret_cast<v4u *>(p) = vpack<T>(f);
    } else if constexpr (VEC) {
        store4<T>(p, f[0], f[1], f[2], f[3]);
    } else {
#pragma unroll
        for (int k = 0; k < V; ++k)
            if (k < cleft) p[k] = from_f32<T>(f[k]);
    }
}

// Workgroups are dispatched round-robin over the 8 XCDs, each with its own
// L2: renumber so that each XCD takes a contiguous range of logical blocks
// (neighbouring pixel chunks share the halo rows of the filter).
__device__ __forceinline__ int dw_logical_block(int id, int total) {
    const int q = total >> 3;
    return id < (q << 3) ? (id & 7) * q + (id >> 3) : id;
}

// Filters of channels c0 .. c0 + CB of the first NTM terms as fp32 [term][tap][channel].
template <typename T, int NTM, int TAPS>
__device__ __forceinline__ void dw_stage_slice(const DwArgs &a, int c0, int CB, float *wl) {
    for (int i = threadIdx.x; i < NTM * TAPS * CB; i += kThreads) {
        const int t = i / (TAPS * CB), rem = i - t * TAPS * CB;
        const int tap = rem / CB, cl = rem - tap * CB;
        const int c = c0 + cl;
        wl[i] = c < a.C ? to_f32<T>(static_cast<const T *>(a.w[t])[(size_t)c * TAPS + tap]) : 0.0f;
    }
}

// acc[k] += w[k] * v[k] over V channels, w the LDS filter row at float offset off (off % 4 == 0).
template <int V>
__device__ __forceinline__ void dw_fma_row(const float *lds, int off, const float *v, float *acc) {
    const float4 *p = reinterpret_cast<const float4 *>(lds) + (off >> 2);
#pragma unroll
    for (int k4 = 0; k4 < V; k4 += 4) {
        const float4 w = p[k4 >> 2];
        acc[k4 + 0] += w.x * v[k4 + 0];
        acc[k4 + 1] += w.y * v[k4 + 1];
        acc[k4 + 2] += w.z * v[k4 + 2];
        acc[k4 + 3] += w.w * v[k4 + 3];
    }
}

// The 3 x 3 kernels loop over chunks of work: the grid holds a fixed number of
// workgroups per channel slice (gridDim.x = tiles x blocks per slice), each
// stages its slice's filters once and takes a contiguous range of chunks of
// `step` work items (a.M items in all).
__device__ __forceinline__ void dw_chunk_range(const DwArgs &a, int step, int &tile, int &ch_begin, int &ch_end) {
    const int lb = dw_logical_block(blockIdx.x, gridDim.x);
    const int nb = gridDim.x / a.tiles;
    tile = lb % a.tiles;
    const int bi = lb / a.tiles;
    const int chunks = (a.M + step - 1) / step;
    const int per = (chunks + nb - 1) / nb;
    ch_begin = bi * per;
    ch_end = min(chunks, ch_begin + per);
}

// Buffer resource of a tensor of `bytes` bytes: a load at an offset past it
// returns zeros, which is how out-of-range taps read 0.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t dw_rsrc(const void *p, int bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, bytes, 0x00020000);
}
constexpr uint32_t kDwOOB = 0x80000000u;  // a byte offset past every tensor the kernels take

// V channels as loaded, converted to fp32 at use (bf16 stays packed in
// registers until then).  VEC: one 16- or 8-byte buffer load at element
// offset `eoff` (zeros when !ok); else element loads through `p`.
template <typename T, int V, bool VEC>
struct DwRaw {
    float f[V];
    __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t, const T *p, int eoff, int cleft, bool ok) {
#pragma unroll
        for (int k = 0; k < V; ++k) f[k] = (ok && k < cleft) ? to_f32<T>(p[(size_t)(unsigned)eoff + k]) : 0.0f;
    }
    __device__ __forceinline__ float get(int k) const { return f[k]; }
};
template <typename T, int V>
struct DwRaw<T, V, true> {
    static constexpr int B = V * (int)sizeof(T);
    static_assert(B == 16 || B == 8, "16- or 8-byte channel vectors");
    typedef typename std::conditional<B == 16, v4u, v2u>::type R;
    R r;
    __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t rs, const T *, int eoff, int, bool ok) {
        const uint32_t bo = ok ? (uint32_t)eoff * (uint32_t)sizeof(T) : kDwOOB;
        if constexpr (B == 16) r = __builtin_amdgcn_raw_buffer_load_b128(rs, bo, 0, 0);
        else r = __builtin_amdgcn_raw_buffer_load_b64(rs, bo, 0, 0);
    }
    __device__ __forceinline__ float get(int k) const {
        if constexpr (sizeof(T) == 4) return __uint_as_float(r[k]);
        else return __uint_as_float((k & 1) ? (r[k >> 1] & 0xffff0000u) : (r[k >> 1] << 16));
    }
};

// V filter (or bias) values at float offset `off` of LDS (off % 4 == 0).
template <int V>
__device__ __forceinline__ void dw_lds_row(const float *lds, int off, float *v) {
    const float4 *p = reinterpret_cast<const float4 *>(lds) + (off >> 2);
#pragma unroll
    for (int k4 = 0; k4 < V / 4; ++k4) {
        const float4 w = p[k4];
        v[4 * k4 + 0] = w.x; v[4 * k4 + 1] = w.y; v[4 * k4 + 2] = w.z; v[4 * k4 + 3] = w.w;
    }
}

// The biases of the slice as fp32 [term][c] (forward).
template <int NTM>
__device__ __forceinline__ void dw_stage_bias(const DwArgs &a, int c0, int CB, float *bl) {
    for (int i = threadIdx.x; i < NTM * CB; i += kThreads) {
        const int t = i / CB, c = c0 + i - t * CB;
        bl[i] = (a.bias[t] && c < a.C) ? a.bias[t][c] : 0.0f;
    }
}

// A compiler fence at the top of each chunk: the filter values are then read
// from LDS within the chunk instead of being hoisted out of the chunk loop
// into registers (27 V of them), which would bound the occupancy.
#define QL_DW_CHUNK_FENCE() asm volatile("" ::: "memory")

// One column of the forward: its position and the raw input rows it sees.
template <typename T, int V, bool VEC, int K, int S, int R>
struct DwFwdCol {
    static constexpr int NIR = (R - 1) * S + K;
    DwRaw<T, V, VEC> xr[NIR][K];
    int item, n, oh0, ow;

    __device__ __forceinline__ void fetch(const DwArgs &a, __amdgpu_buffer_rsrc_t xrs, const T *x, int it_, int c,
                                          int cleft) {
        item = it_;
        const int it = min(it_, a.M - 1);  // past the end: a valid column, loaded but not stored
        n = (int)fdiv((uint32_t)it, a.fd_item);
        const int rem = it - n * a.ng * a.iwid;
        const int g = (int)fdiv((uint32_t)rem, a.fd_iw);
        ow = rem - g * a.iwid;
        oh0 = g * R;
        const int ih0 = oh0 * S - a.PH, iw0 = ow * S - a.PW;
        const int base = ((n * a.H + ih0) * a.W + iw0) * a.C + c;  // element offset of tap (0, 0)
        const int rowc = a.W * a.C;
#pragma unroll
        for (int ir = 0; ir < NIR; ++ir) {
            const bool okr = (unsigned)(ih0 + ir) < (unsigned)a.H;
#pragma unroll
            for (int q = 0; q < K; ++q) {
                const bool ok = okr && (unsigned)(iw0 + q) < (unsigned)a.W;
                xr[ir][q].load(xrs, x, base + ir * rowc + q * a.C, cleft, ok);
            }
        }
    }
};

// Forward, K x K at stride S, by columns: a thread takes V channels of R
// consecutive output rows of one output column, (R - 1) S + K input rows of
// K columns loaded once, and each filter value read from LDS serves the R
// rows.  PF: the next column's loads are issued before the current column's
// arithmetic (two register buffers).  a.M counts the columns N x ceil(HO / R) x WO.
template <typename T, int OM, int V, bool VEC, int K, int S, int R>
__device__ __forceinline__ void dw_fwd_col_compute(const DwArgs &a, const DwFwdCol<T, V, VEC, K, S, R> &b,
                                                   const float *wl, const float *bl, int CB, int cg, int c,
                                                   int cleft) {
    constexpr int NTM = om_terms(OM), TAPS = K * K;
    if (b.item >= a.M) return;
    const T *__restrict__ x = static_cast<const T *>(a.x);
    float acc[R][NTM][V];
#pragma unroll
    for (int t = 0; t < NTM; ++t) {
        float bv[V];
        dw_lds_row<V>(bl, t * CB + V * cg, bv);
#pragma unroll
        for (int rr = 0; rr < R; ++rr)
#pragma unroll
            for (int k = 0; k < V; ++k) acc[rr][t][k] = bv[k];
    }
#pragma unroll
    for (int r = 0; r < K; ++r) {
#pragma unroll
        for (int q = 0; q < K; ++q) {
            float xs[R][V];
#pragma unroll
            for (int rr = 0; rr < R; ++rr)
#pragma unroll
                for (int k = 0; k < V; ++k) {
                    const float v = b.xr[rr * S + r][q].get(k);
                    xs[rr][k] = OM == OM_SQIN ? to_f32<T>(from_f32<T>(v * v)) : v;  // T2: X o X in T
                }
#pragma unroll
            for (int t = 0; t < NTM; ++t) {
                float wv[V];
                dw_lds_row<V>(wl, (t * TAPS + r * K + q) * CB + V * cg, wv);
#pragma unroll
                for (int rr = 0; rr < R; ++rr)
#pragma unroll
                    for (int k = 0; k < V; ++k) acc[rr][t][k] += wv[k] * xs[rr][k];
            }
        }
    }
#pragma unroll
    for (int rr = 0; rr < R; ++rr) {
        if (b.oh0 + rr >= a.HO) break;
        const size_t off = ((size_t)(b.n * a.HO + b.oh0 + rr) * a.WO + b.ow) * a.C + c;
        float yv[V];
        float xs[V];
        if (OM == OM_PAIR && a.neuron == NEURON_T4I) {
            dw_ldv<T, V, VEC>(x + off, cleft, xs);  // the same pixel of X (the map keeps its size)
        } else {
#pragma unroll
            for (int k = 0; k < V; ++k) xs[k] = 0.0f;
        }
#pragma unroll
        for (int k = 0; k < V; ++k) {
            const float fa = acc[rr][0][k];
            if constexpr (OM == OM_QUADRA) yv[k] = fa * acc[rr][1][k] + acc[rr][2][k];
            else if constexpr (OM == OM_PAIR) yv[k] = fa * acc[rr][1][k] + xs[k];
            else if constexpr (OM == OM_SQUARE) yv[k] = fa * fa;
            else yv[k] = fa;
            if (k < cleft) yv[k] = epi_apply(a.epi, c + k, yv[k]);
        }
        if (a.y) dw_stv<T, V, VEC>(static_cast<T *>(a.y) + off, cleft, yv);
        if (a.yta) dw_stv<T, V, VEC>(static_cast<T *>(a.yta) + off, cleft, acc[rr][0]);
        if constexpr (NTM >= 2) {
            if (a.ytb) dw_stv<T, V, VEC>(static_cast<T *>(a.ytb) + off, cleft, acc[rr][1]);
        }
    }
}

template <typename T, int OM, int V, bool VEC, int K, int S, int R, bool PF>
__global__ __launch_bounds__(kThreads)
void qconv_dw_fwd_col_kernel(const DwArgs a) {
    constexpr int NTM = om_terms(OM), TAPS = K * K;
    extern __shared__ float wl[];  // [NTM][TAPS][CB], then the biases [NTM][CB]
    const int CB = a.lanes * V;
    const int cg = threadIdx.x & (a.lanes - 1), pl = threadIdx.x >> a.lsh, PL = kThreads >> a.lsh;
    int tile, ch_begin, ch_end;
    dw_chunk_range(a, PL, tile, ch_begin, ch_end);
    const int c0 = tile * CB;
    float *bl = wl + NTM * TAPS * CB;
    dw_stage_slice<T, NTM, TAPS>(a, c0, CB, wl);
    dw_stage_bias<NTM>(a, c0, CB, bl);
    __syncthreads();
    const int c = c0 + V * cg, cleft = a.C - c;
    if (cleft <= 0 || ch_begin >= ch_end) return;
    const T *__restrict__ x = static_cast<const T *>(a.x);
    const __amdgpu_buffer_rsrc_t xrs = dw_rsrc(a.x, a.xbytes);
    if constexpr (!PF) {
        for (int chunk = ch_begin; chunk < ch_end; ++chunk) {
            QL_DW_CHUNK_FENCE();
            DwFwdCol<T, V, VEC, K, S, R> b;
            b.fetch(a, xrs, x, chunk * PL + pl, c, cleft);
            dw_fwd_col_compute<T, OM>(a, b, wl, bl, CB, cg, c, cleft);
        }
        return;
    }
    DwFwdCol<T, V, VEC, K, S, R> b0, b1;
    int chunk = ch_begin;
    b0.fetch(a, xrs, x, chunk * PL + pl, c, cleft);
    // the next fetch is unconditional (clamped, not stored past the end): no
    // branch between a fetch and its use
    while (true) {
        QL_DW_CHUNK_FENCE();
        b1.fetch(a, xrs, x, (chunk + 1) * PL + pl, c, cleft);
        dw_fwd_col_compute<T, OM>(a, b0, wl, bl, CB, cg, c, cleft);
        if (++chunk >= ch_end) break;
        QL_DW_CHUNK_FENCE();
        b0.fetch(a, xrs, x, (chunk + 1) * PL + pl, c, cleft);
        dw_fwd_col_compute<T, OM>(a, b1, wl, bl, CB, cg, c, cleft);
        if (++chunk >= ch_end) break;
    }
}

// The output-side operands of the neuron type at one output pixel, V channels:
// QUADRA: G o T_b, G o T_a, G; PAIR: G o T_b, G o T_a; SQUARE: 2 G o T_a; SQIN: G.
template <int OM, int V, typename Raw>
__device__ __forceinline__ void dw_ops(const Raw *gv, float (*op)[V]) {
#pragma unroll
    for (int k = 0; k < V; ++k) {
        const float g = gv[0].get(k);
        if constexpr (OM == OM_QUADRA || OM == OM_PAIR) {
            op[0][k] = g * gv[2].get(k);
            op[1][k] = g * gv[1].get(k);
            if constexpr (OM == OM_QUADRA) op[2][k] = g;
        } else if constexpr (OM == OM_SQUARE) {
            op[0][k] = 2.0f * g * gv[1].get(k);
        } else {
            op[0][k] = g;
        }
    }
}

// Input-gradient epilogue at input pixel offset `off`: T2 multiplies by 2 X
// (X arrives in `ta`), T4 + identity adds G at the same pixel.
template <typename T, int OM, int V, bool VEC>
__device__ __forceinline__ void dw_dx_store(const DwArgs &a, size_t off, int cleft, float *acc) {
    if (OM == OM_SQIN || (OM == OM_PAIR && a.neuron == NEURON_T4I)) {
        float v[V];
        dw_ldv<T, V, VEC>(static_cast<const T *>(OM == OM_SQIN ? a.ta : a.gy) + off, cleft, v);
#pragma unroll
        for (int k = 0; k < V; ++k) acc[k] = OM == OM_SQIN ? acc[k] * (2.0f * v[k]) : acc[k] + v[k];
    }
    dw_stv<T, V, VEC>(static_cast<T *>(a.dx) + off, cleft, acc);
}

// One column of the stride-1 input gradient: its position and the raw
// output-side maps of the R + K - 1 output rows it needs.
template <typename T, int OM, int V, bool VEC, int K, int R>
struct DwBdCol {
    static constexpr int NGM = om_gmaps(OM), NOR = R + K - 1;
    DwRaw<T, V, VEC> gv[NOR][K][NGM];
    int item, n, h0, w;

    __device__ __forceinline__ void fetch(const DwArgs &a, const __amdgpu_buffer_rsrc_t *mrs, const T *const *maps,
                                          int it_, int c, int cleft) {
        item = it_;
        const int it = min(it_, a.M - 1);
        n = (int)fdiv((uint32_t)it, a.fd_item);
        const int rem = it - n * a.ng * a.iwid;
        const int g = (int)fdiv((uint32_t)rem, a.fd_iw);
        w = rem - g * a.iwid;
        h0 = g * R;
        const int oi0 = h0 + a.PH - (K - 1), oj0 = w + a.PW;
        const int base = ((n * a.HO + oi0) * a.WO + oj0) * a.C + c;  // output row oi0, column oj0
        const int rowc = a.WO * a.C;
#pragma unroll
        for (int e = 0; e < NOR; ++e) {
            const bool okr = (unsigned)(oi0 + e) < (unsigned)a.HO;
#pragma unroll
            for (int q = 0; q < K; ++q) {
                const bool ok = okr && (unsigned)(oj0 - q) < (unsigned)a.WO;
#pragma unroll
                for (int m = 0; m < NGM; ++m) gv[e][q][m].load(mrs[m], maps[m], base + e * rowc - q * a.C, cleft, ok);
            }
        }
    }
};

template <typename T, int OM, int V, bool VEC, int K, int R>
__device__ __forceinline__ void dw_bd_col_compute(const DwArgs &a, const DwBdCol<T, OM, V, VEC, K, R> &b,
                                                  const float *wl, int CB, int cg, int c, int cleft) {
    constexpr int NTM = om_terms(OM), TAPS = K * K, NOR = R + K - 1;
    if (b.item >= a.M) return;
    float acc[R][V];
#pragma unroll
    for (int rr = 0; rr < R; ++rr)
#pragma unroll
        for (int k = 0; k < V; ++k) acc[rr][k] = 0.0f;
#pragma unroll
    for (int e = 0; e < NOR; ++e) {
#pragma unroll
        for (int q = 0; q < K; ++q) {
            float op[3][V];
            dw_ops<OM, V>(b.gv[e][q], op);
#pragma unroll
            for (int rr = 0; rr < R; ++rr) {
                const int r = rr + (K - 1) - e;  // the tap input row h0 + rr takes from this output row
                if (r < 0 || r >= K) continue;
#pragma unroll
                for (int t = 0; t < NTM; ++t) dw_fma_row<V>(wl, (t * TAPS + r * K + q) * CB + V * cg, op[t], acc[rr]);
            }
        }
    }
#pragma unroll
    for (int rr = 0; rr < R; ++rr) {
        if (b.h0 + rr >= a.H) break;
        dw_dx_store<T, OM, V, VEC>(a, ((size_t)(b.n * a.H + b.h0 + rr) * a.W + b.w) * a.C + c, cleft, acc[rr]);
    }
}

// Input gradient, K x K at stride 1, by columns: a thread takes V channels of
// R consecutive input rows of one input column; input row h takes tap r from
// output row h + p - r, so the column needs R + K - 1 output rows, whose
// operands are formed once per row and applied to every input row they feed.
// PF: the next column's loads are issued before the current column's
// arithmetic.  a.M counts the columns N x ceil(H / R) x W.
template <typename T, int OM, int V, bool VEC, int K, int R, bool PF>
__global__ __launch_bounds__(kThreads)
void qconv_dw_bwd_data_col_kernel(const DwArgs a) {
    constexpr int NTM = om_terms(OM), NGM = om_gmaps(OM), TAPS = K * K;
    extern __shared__ float wl[];
    const int CB = a.lanes * V;
    const int cg = threadIdx.x & (a.lanes - 1), pl = threadIdx.x >> a.lsh, PL = kThreads >> a.lsh;
    int tile, ch_begin, ch_end;
    dw_chunk_range(a, PL, tile, ch_begin, ch_end);
    const int c0 = tile * CB;
    dw_stage_slice<T, NTM, TAPS>(a, c0, CB, wl);
    __syncthreads();
    const int c = c0 + V * cg, cleft = a.C - c;
    if (cleft <= 0 || ch_begin >= ch_end) return;
    const T *maps[3] = {static_cast<const T *>(a.gy), static_cast<const T *>(a.ta), static_cast<const T *>(a.tb)};
    __amdgpu_buffer_rsrc_t mrs[3];
#pragma unroll
    for (int m = 0; m < NGM; ++m) mrs[m] = dw_rsrc(maps[m], a.pbytes);
    if constexpr (!PF) {
        for (int chunk = ch_begin; chunk < ch_end; ++chunk) {
            QL_DW_CHUNK_FENCE();
            DwBdCol<T, OM, V, VEC, K, R> b;
            b.fetch(a, mrs, maps, chunk * PL + pl, c, cleft);
            dw_bd_col_compute<T, OM, V, VEC, K, R>(a, b, wl, CB, cg, c, cleft);
        }
        return;
    }
    DwBdCol<T, OM, V, VEC, K, R> b0, b1;
    int chunk = ch_begin;
    b0.fetch(a, mrs, maps, chunk * PL + pl, c, cleft);
    while (true) {
        QL_DW_CHUNK_FENCE();
        b1.fetch(a, mrs, maps, (chunk + 1) * PL + pl, c, cleft);
        dw_bd_col_compute<T, OM, V, VEC, K, R>(a, b0, wl, CB, cg, c, cleft);
        if (++chunk >= ch_end) break;
        QL_DW_CHUNK_FENCE();
        b0.fetch(a, mrs, maps, (chunk + 1) * PL + pl, c, cleft);
        dw_bd_col_compute<T, OM, V, VEC, K, R>(a, b1, wl, CB, cg, c, cleft);
        if (++chunk >= ch_end) break;
    }
}

// Input gradient, K x K at stride S (any), by gathering: input row h takes tap
// r from output row (h + p - r) / S when S divides h + p - r, so only r =
// (h + p) mod S + S t, t < ceil(K / S), are gathered (likewise q); the
// others read the zero page.  One input pixel of V channels per thread and
// chunk; a.M counts the input pixels.
template <typename T, int OM, int V, bool VEC, int K, int S>
__global__ __launch_bounds__(kThreads)
void qconv_dw_bwd_data_k_kernel(const DwArgs a) {
    constexpr int NTM = om_terms(OM), NGM = om_gmaps(OM), TAPS = K * K, NR = (K + S - 1) / S;
    extern __shared__ float wl[];
    const int CB = a.lanes * V;
    const int cg = threadIdx.x & (a.lanes - 1), pl = threadIdx.x >> a.lsh, PL = kThreads >> a.lsh;
    int tile, ch_begin, ch_end;
    dw_chunk_range(a, PL, tile, ch_begin, ch_end);
    const int c0 = tile * CB;
    dw_stage_slice<T, NTM, TAPS>(a, c0, CB, wl);
    __syncthreads();
    const int c = c0 + V * cg, cleft = a.C - c;
    if (cleft <= 0) return;
    const T *maps[3] = {static_cast<const T *>(a.gy), static_cast<const T *>(a.ta), static_cast<const T *>(a.tb)};
    __amdgpu_buffer_rsrc_t mrs[3];
#pragma unroll
    for (int m = 0; m < NGM; ++m) mrs[m] = dw_rsrc(maps[m], a.pbytes);
    for (int chunk = ch_begin; chunk < ch_end; ++chunk) {
        QL_DW_CHUNK_FENCE();
        const int mm = chunk * PL + pl;
        const int m = min(mm, a.M - 1);
        const int n = (int)fdiv((uint32_t)m, a.fd_hw);
        const int rem = m - n * a.H * a.W;
        const int h = (int)fdiv((uint32_t)rem, a.fd_w);
        const int w = rem - h * a.W;
        const int hr = h + a.PH, wr = w + a.PW;
        const int r0 = hr % S, q0 = wr % S;
        DwRaw<T, V, VEC> gv[NR * NR][NGM];
        int tapi[NR * NR];
#pragma unroll
        for (int tr = 0; tr < NR; ++tr) {
            const int r = r0 + S * tr;
            const int i = (hr - r) / S;  // exact when r <= hr
            const bool okr = r < K && r <= hr && i < a.HO;
#pragma unroll
            for (int tq = 0; tq < NR; ++tq) {
                const int q = q0 + S * tq;
                const int j = (wr - q) / S;
                const bool ok = okr && q < K && q <= wr && j < a.WO;
                const int slot = tr * NR + tq;
                tapi[slot] = ok ? r * K + q : 0;
                const int go = ((n * a.HO + i) * a.WO + j) * a.C + c;
#pragma unroll
                for (int g = 0; g < NGM; ++g) gv[slot][g].load(mrs[g], maps[g], go, cleft, ok);
            }
        }
        float acc[V];
#pragma unroll
        for (int k = 0; k < V; ++k) acc[k] = 0.0f;
#pragma unroll
        for (int slot = 0; slot < NR * NR; ++slot) {
            float op[3][V];
            dw_ops<OM, V>(gv[slot], op);
#pragma unroll
            for (int t = 0; t < NTM; ++t) dw_fma_row<V>(wl, (t * TAPS + tapi[slot]) * CB + V * cg, op[t], acc);
        }
        if (mm >= a.M) continue;
        dw_dx_store<T, OM, V, VEC>(a, (size_t)mm * a.C + c, cleft, acc);
    }
}

// Weight and bias gradients, K x K at stride S, by columns: a block takes one
// channel slice (lanes x V channels) and one split of the columns (image,
// row group of R output rows, output column); a thread accumulates every tap
// of its channels over its columns: the operands of R output pixels and the
// (R - 1) S + K rows of K input columns they see, loaded once per column.
// The loads of the next column are issued before the arithmetic of the
// current one (two register buffers, raw until use).  The pixel lanes are
// then summed in a fixed order through LDS.  a.M counts the columns.
template <typename T, int OM, int V, bool VEC, int K, int S, int R>
struct DwBwCol {
    static constexpr int NGM = om_gmaps(OM), NIR = (R - 1) * S + K;
    DwRaw<T, V, VEC> gv[R][NGM], xr[NIR][K];

    __device__ __forceinline__ void fetch(const DwArgs &a, const __amdgpu_buffer_rsrc_t *mrs, const T *const *maps,
                                          __amdgpu_buffer_rsrc_t xrs, const T *x, int item, int i_end, int c,
                                          int cleft) {
        const bool live = item < i_end;
        const int it = min(item, a.M - 1);
        const int n = (int)fdiv((uint32_t)it, a.fd_item);
        const int rem = it - n * a.ng * a.iwid;
        const int g = (int)fdiv((uint32_t)rem, a.fd_iw);
        const int ow = rem - g * a.iwid;
        const int oh0 = g * R;
        const int gbase = ((n * a.HO + oh0) * a.WO + ow) * a.C + c;
#pragma unroll
        for (int rr = 0; rr < R; ++rr) {
            const bool ok = live && oh0 + rr < a.HO;  // rows past the map, columns past the split: zero operands
#pragma unroll
            for (int m = 0; m < NGM; ++m) gv[rr][m].load(mrs[m], maps[m], gbase + rr * a.WO * a.C, cleft, ok);
        }
        const int ih0 = oh0 * S - a.PH, iw0 = ow * S - a.PW;
        const int xbase = ((n * a.H + ih0) * a.W + iw0) * a.C + c;
#pragma unroll
        for (int ir = 0; ir < NIR; ++ir) {
            const bool okr = (unsigned)(ih0 + ir) < (unsigned)a.H;
#pragma unroll
            for (int q = 0; q < K; ++q) {
                const bool ok = okr && (unsigned)(iw0 + q) < (unsigned)a.W;
                xr[ir][q].load(xrs, x, xbase + (ir * a.W + q) * a.C, cleft, ok);
            }
        }
    }

    template <int NTM>
    __device__ __forceinline__ void consume(float (&acc)[NTM][K * K][V], float (&dsum)[NTM][V]) const {
        float op[R][3][V];
#pragma unroll
        for (int rr = 0; rr < R; ++rr) {
            dw_ops<OM, V>(gv[rr], op[rr]);
#pragma unroll
            for (int t = 0; t < NTM; ++t)
#pragma unroll
                for (int k = 0; k < V; ++k) dsum[t][k] += op[rr][t][k];
        }
#pragma unroll
        for (int r = 0; r < K; ++r)
#pragma unroll
            for (int q = 0; q < K; ++q)
#pragma unroll
                for (int rr = 0; rr < R; ++rr)
#pragma unroll
                    for (int k = 0; k < V; ++k) {
                        const float v = xr[rr * S + r][q].get(k);
                        const float xs = OM == OM_SQIN ? to_f32<T>(from_f32<T>(v * v)) : v;
#pragma unroll
                        for (int t = 0; t < NTM; ++t) acc[t][r * K + q][k] += op[rr][t][k] * xs;
                    }
    }
};

template <typename T, int OM, int V, bool VEC, int K, int S, int R>
__global__ __launch_bounds__(kThreads)
void qconv_dw_bwd_weight_col_kernel(const DwArgs a) {
    constexpr int NTM = om_terms(OM), TAPS = K * K;
    __shared__ float wsum[(kThreads / 64) * 8 * NTM * (TAPS + 1) * V];  // [wave][channel group][...]
    const int CB = a.lanes * V;
    const int split = blockIdx.x, c0 = blockIdx.y * CB;
    const int cg = threadIdx.x & (a.lanes - 1), pl = threadIdx.x >> a.lsh, PL = kThreads >> a.lsh;
    const int c = c0 + V * cg, cleft = a.C - c;
    const int i_begin = split * a.px_per_split, i_end = min(a.M, i_begin + a.px_per_split);
    const T *__restrict__ x = static_cast<const T *>(a.x);
    const T *maps[3] = {static_cast<const T *>(a.gy), static_cast<const T *>(a.ta), static_cast<const T *>(a.tb)};
    constexpr int NGM = om_gmaps(OM);
    __amdgpu_buffer_rsrc_t mrs[3];
#pragma unroll
    for (int m = 0; m < NGM; ++m) mrs[m] = dw_rsrc(maps[m], a.pbytes);
    const __amdgpu_buffer_rsrc_t xrs = dw_rsrc(a.x, a.xbytes);
    float acc[NTM][TAPS][V], dsum[NTM][V];
#pragma unroll
    for (int t = 0; t < NTM; ++t) {
#pragma unroll
        for (int k = 0; k < V; ++k) dsum[t][k] = 0.0f;
#pragma unroll
        for (int u = 0; u < TAPS; ++u)
#pragma unroll
            for (int k = 0; k < V; ++k) acc[t][u][k] = 0.0f;
    }
    if (cleft > 0 && i_begin + pl < i_end) {
        DwBwCol<T, OM, V, VEC, K, S, R> b0, b1;
        int item = i_begin + pl;
        b0.fetch(a, mrs, maps, xrs, x, item, i_end, c, cleft);
        // the next fetch is unconditional (clamped, dead columns read zeros):
        // no branch between a fetch and its use
        while (true) {
            b1.fetch(a, mrs, maps, xrs, x, item + PL, i_end, c, cleft);
            b0.template consume<NTM>(acc, dsum);
            item += PL;
            if (item >= i_end) break;
            b0.fetch(a, mrs, maps, xrs, x, item + PL, i_end, c, cleft);
            b1.template consume<NTM>(acc, dsum);
            item += PL;
            if (item >= i_end) break;
        }
    }
    // Sum over the pixel lanes in a fixed order: a butterfly over the lanes of
    // each wave that share the channel group (lane bits lsh .. 5; every
    // value's exchange of one step issued together), then the four waves in
    // wave order through LDS.
    constexpr int NV = NTM * (TAPS + 1) * V;  // per thread: every tap, then the bias sum
    for (int m = a.lanes; m < 64; m <<= 1) {
#pragma unroll
        for (int t = 0; t < NTM; ++t)
#pragma unroll
            for (int k = 0; k < V; ++k) {
#pragma unroll
                for (int u = 0; u < TAPS; ++u) acc[t][u][k] += __shfl_xor(acc[t][u][k], m);
                dsum[t][k] += __shfl_xor(dsum[t][k], m);
            }
    }
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    if (lane < a.lanes) {  // one lane per channel group and wave holds the wave's sums
        float *r = wsum + (wave * 8 + cg) * NV;
#pragma unroll
        for (int t = 0; t < NTM; ++t)
#pragma unroll
            for (int k = 0; k < V; ++k) {
#pragma unroll
                for (int u = 0; u < TAPS; ++u) r[(t * (TAPS + 1) + u) * V + k] = acc[t][u][k];
                r[(t * (TAPS + 1) + TAPS) * V + k] = dsum[t][k];
            }
    }
    __syncthreads();
    // output (t, u, channel c0 + cc) for u < TAPS a weight tap, u = TAPS the bias
    for (int i = threadIdx.x; i < NTM * (TAPS + 1) * CB; i += kThreads) {
        const int t = i / ((TAPS + 1) * CB), rem = i - t * (TAPS + 1) * CB;
        const int u = rem / CB, cc = rem - u * CB;
        const int g2 = cc / V, k = cc - g2 * V;
        const int ch = c0 + cc;
        if (ch >= a.C || (u == TAPS && !a.db[t])) continue;
        float sum = 0.0f;
#pragma unroll
        for (int w = 0; w < kThreads / 64; ++w) sum += wsum[(w * 8 + g2) * NV + (t * (TAPS + 1) + u) * V + k];
        float *dst;
        if (u < TAPS)
            dst = a.splits == 1 ? a.dw[t] + (size_t)ch * TAPS + u
                                : a.ws + (size_t)split * a.J + ((size_t)t * a.C + ch) * TAPS + u;
        else
            dst = a.splits == 1 ? a.db[t] + ch : a.ws + (size_t)split * a.J + (size_t)(NTM * TAPS + t) * a.C + ch;
        *dst = sum;
    }
}

}  // namespace ql
