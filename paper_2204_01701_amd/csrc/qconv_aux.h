// qconv_aux.h -- auxiliary kernels of the quadratic layer: the split-K
// epilogue of the forward, the split-K reductions of the gradients (all in
// split order, so results are deterministic) and the per-term weight
// transpose used by the fp32 input gradient.  Grid-stride loops over 4
// consecutive elements when the innermost extent allows 16-byte accesses.
#pragma once

#include "qdevice.h"

namespace ql {

// Forward split-K epilogue: T_t = b_t + sum over splits of the partials, then
// Y = T_a o T_b + T_c (arXiv 2204.01701, eq:2ndneuron3; for T2&4 the partials
// of T_c are already those of W_c (X o X)) or the neuron type's Y.  ws: [split][3][M*O].
template <typename T, bool V4>
__global__ __launch_bounds__(kThreads) void qconv_fwd_combine_kernel(const float *__restrict__ ws, int splits,
                                                                     long long MO, int O, const float *b0,
                                                                     const float *b1, const float *b2, T *y, T *ta,
                                                                     T *tb, int neuron, const T *x, EpiArgs epi) {
    constexpr int E = V4 ? 4 : 1;
    const float *bp[3] = {b0, b1, b2};
    const bool three = neuron == NEURON_QUADRA || neuron == NEURON_T24;  // (T2&4: T_c already on X o X)
    const int nt = three ? 3 : (neuron <= NEURON_T4I ? 2 : 1);
    const long long n = MO / E;
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (long long)gridDim.x * blockDim.x) {
        const long long idx = i * E;
        const int o = (int)(idx % O);
        float t3[3][E];
#pragma unroll
        for (int t = 0; t < 3; ++t) {
#pragma unroll
            for (int e = 0; e < E; ++e) t3[t][e] = (t < nt && bp[t]) ? bp[t][o + e] : 0.0f;
            if (t >= nt) continue;
#pragma unroll 4
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
        // the layer output of the neuron type (the shortcut of T4 + identity: C == O, same pixel)
        float yv[E];
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const float fa = t3[0][e], fb = t3[1][e];
            if (three) yv[e] = fa * fb + t3[2][e];
            else if (neuron == NEURON_T4) yv[e] = fa * fb;
            else if (neuron == NEURON_T4I) yv[e] = fa * fb + to_f32<T>(x[idx + e]);
            else if (neuron == NEURON_T3) yv[e] = fa * fa;
            else yv[e] = fa;
            yv[e] = epi_apply(epi, o + e, yv[e]);
        }
        if (nt < 2) tb = nullptr;
        if constexpr (V4) {
            if (y) store4<T>(y + idx, yv[0], yv[1], yv[2], yv[3]);
            if (ta) store4<T>(ta + idx, t3[0][0], t3[0][1], t3[0][2], t3[0][3]);
            if (tb) store4<T>(tb + idx, t3[1][0], t3[1][1], t3[1][2], t3[1][3]);
        } else {
            if (y) y[idx] = from_f32<T>(yv[0]);
            if (ta) ta[idx] = from_f32<T>(t3[0][0]);
            if (tb) tb[idx] = from_f32<T>(t3[1][0]);
        }
    }
}

// Sum of `splits` partial buffers of `total` floats each, in split order; the
// result is converted to T.  mode 1 adds src (the shortcut gradient G of
// T4 + identity), mode 2 multiplies by 2 src (X for T2); src has `total` elements.
template <typename T, bool V4>
__global__ __launch_bounds__(kThreads) void qconv_sum_splits_kernel(const float *__restrict__ ws, int splits,
                                                                    long long total, T *__restrict__ out, int mode,
                                                                    const T *__restrict__ src) {
    constexpr int E = V4 ? 4 : 1;
    const long long n = total / E;
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (long long)gridDim.x * blockDim.x) {
        const long long idx = i * E;
        float acc[E];
#pragma unroll
        for (int e = 0; e < E; ++e) acc[e] = 0.0f;
#pragma unroll 4
        for (int sp = 0; sp < splits; ++sp) {
            const float *p = ws + (size_t)sp * total + idx;
            if constexpr (V4) {
                const v4f v = *reinterpret_cast<const v4f *>(p);
#pragma unroll
                for (int e = 0; e < 4; ++e) acc[e] += v[e];
            } else {
                acc[0] += p[0];
            }
        }
        if (mode != 0) {
#pragma unroll
            for (int e = 0; e < E; ++e) {
                const float v = to_f32<T>(src[idx + e]);
                acc[e] = mode == 1 ? acc[e] + v : acc[e] * (2.0f * v);
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
                                                                           int want_db, int nterms) {
    constexpr int E = V4 ? 4 : 1;
    const long long nv = nterms * ndw / E;
    const long long total = nv + (want_db ? (long long)nterms * O : 0LL);
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (long long)gridDim.x * blockDim.x) {
        if (i < nv) {
            const long long idx = i * E;
            const int t = (int)(idx / ndw);
            const long long j = idx - t * ndw;
            float acc[E];
#pragma unroll
            for (int e = 0; e < E; ++e) acc[e] = 0.0f;
#pragma unroll 4
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

// The same reduction for small outputs with many splits, 16-byte vectors
// (ndw % 4 == 0): a block takes 16 items (an item is 4 consecutive dW_t
// values, or one bias value after the nterms ndw / 4 vectors); 16 split
// lanes per item sum every 16th split (unrolled, the loads independent) and
// the lane sums are added in lane order, the same order as the scalar kernel.
template <int = 0>  // (a template: defined once across the translation units that include this header)
__global__ __launch_bounds__(kThreads) void qconv_bwd_weight_reduce2dv_kernel(const float *__restrict__ ws_dw,
                                                                              const float *__restrict__ ws_db,
                                                                              int splits, long long ndw, int O,
                                                                              float *dw0, float *dw1, float *dw2,
                                                                              float *db0, float *db1, float *db2,
                                                                              int want_db, int nterms) {
    __shared__ v4f part[16][17];
    const long long nv = (long long)nterms * ndw / 4;
    const long long total = nv + (want_db ? (long long)nterms * O : 0LL);
    const int it = threadIdx.x & 15, sl = threadIdx.x >> 4;
    for (long long base = (long long)blockIdx.x * 16; base < total; base += (long long)gridDim.x * 16) {
        const long long i = base + it;
        v4f s = {0.0f, 0.0f, 0.0f, 0.0f};
        if (i < nv) {
            const long long idx = i * 4;
            const int t = (int)(idx / ndw);
            const long long j = idx - t * ndw;
#pragma unroll 4
            for (int sp = sl; sp < splits; sp += 16) s += *reinterpret_cast<const v4f *>(ws_dw + ((size_t)sp * 3 + t) * ndw + j);
        } else if (i < total) {
            const long long jj = i - nv;
            const int t = (int)(jj / O), o = (int)(jj % O);
#pragma unroll 4
            for (int sp = sl; sp < splits; sp += 16) s[0] += ws_db[((size_t)sp * 3 + t) * O + o];
        }
        part[sl][it] = s;
        __syncthreads();
        if (sl == 0 && i < total) {
            v4f acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int k = 0; k < 16; ++k) acc += part[k][it];
            if (i < nv) {
                const long long idx = i * 4;
                const int t = (int)(idx / ndw);
                float *d = t == 0 ? dw0 : (t == 1 ? dw1 : dw2);
                *reinterpret_cast<v4f *>(d + (idx - t * ndw)) = acc;
            } else {
                const long long jj = i - nv;
                const int t = (int)(jj / O), o = (int)(jj % O);
                float *d = t == 0 ? db0 : (t == 1 ? db1 : db2);
                d[o] = acc[0];
            }
        }
        __syncthreads();
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
                                                                             int want_db, int nterms) {
    constexpr int PER = kThreads / SG;
    __shared__ float part[SG][PER];
    const long long nw = (long long)nterms * ndw;
    const long long total = nw + (want_db ? (long long)nterms * O : 0LL);
    const int e = threadIdx.x % PER, sg = threadIdx.x / PER;
    for (long long base = (long long)blockIdx.x * PER; base < total; base += (long long)gridDim.x * PER) {
        const long long i = base + e;
        float s = 0.0f;
        if (i < total) {
            if (i < nw) {
                const int t = (int)(i / ndw);
                const long long j = i - t * ndw;
                for (int sp = sg; sp < splits; sp += SG) s += ws_dw[((size_t)sp * 3 + t) * ndw + j];
            } else {
                const long long jj = i - nw;
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
            if (i < nw) {
                const int t = (int)(i / ndw);
                float *d = t == 0 ? dw0 : (t == 1 ? dw1 : dw2);
                d[i - t * ndw] = acc;
            } else {
                const long long jj = i - nw;
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
// Elementwise X o X (the operand of the T2 neuron), 16 bytes per thread and
// step; n: elements, a multiple of the 16-byte vector.
template <typename T>
__global__ __launch_bounds__(kThreads) void qconv_square_kernel(const T *__restrict__ src, T *__restrict__ dst,
                                                                long long n) {
    constexpr int VEC = Elem<T>::VEC;
    const long long nv = n / VEC;
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < nv; i += (long long)gridDim.x * blockDim.x)
        *reinterpret_cast<v4u *>(dst + i * VEC) = square_frag<T>(*reinterpret_cast<const v4u *>(src + i * VEC));
}

// The ReLU's backward in front of the layer's: out = g where y > 0, else 0
// (y the stored activation y' = relu(Y), g = dl/dy'), so out = dl/dY.  16
// bytes per thread and step, the tail of n past the last whole vector one
// element per thread.  g, y, out 16-byte aligned.
template <typename T>
__global__ __launch_bounds__(kThreads) void qconv_relu_mask_kernel(const T *__restrict__ g, const T *__restrict__ y,
                                                                   T *__restrict__ out, long long n) {
    constexpr int VEC = Elem<T>::VEC;
    const long long nv = n / VEC;
    const long long stride = (long long)gridDim.x * blockDim.x;
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < nv; i += stride) {
        const v4u gv = *reinterpret_cast<const v4u *>(g + i * VEC);
        const v4u yv = *reinterpret_cast<const v4u *>(y + i * VEC);
        float f[VEC];
#pragma unroll
        for (int e = 0; e < VEC; ++e) f[e] = vget<T>(yv, e) > 0.0f ? vget<T>(gv, e) : 0.0f;
        *reinterpret_cast<v4u *>(out + i * VEC) = vpack<T>(f);
    }
    for (long long i = nv * VEC + (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
        out[i] = to_f32(y[i]) > 0.0f ? g[i] : from_f32<T>(0.0f);
}

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
    if (Cp * (int)sizeof(T) == 16) {
        // one padded row per 16-byte store (the usual case: 3 channels padded to 8 bf16 or 4 fp32)
        const long long rows = sg.rows[blockIdx.y];
        for (long long r = (long long)blockIdx.x * blockDim.x + threadIdx.x; r < rows;
             r += (long long)gridDim.x * blockDim.x) {
            float v[16 / sizeof(T)];
#pragma unroll
            for (int c = 0; c < (int)(16 / sizeof(T)); ++c) v[c] = c < C ? to_f32<T>(src[r * C + c]) : 0.0f;
            *reinterpret_cast<v4u *>(dst + r * Cp) = vpack<T>(v);
        }
        return;
    }
    const long long total = sg.rows[blockIdx.y] * Cp;
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (long long)gridDim.x * blockDim.x) {
        const long long r = i / Cp;
        const int c = (int)(i - r * Cp);
        dst[i] = c < C ? src[r * C + c] : T(0);
    }
}

// Input gradient for layers with few input channels (C <= 4, e.g. a network's
// first layer on RGB images).  An MFMA tile with input channels as rows would
// be nearly empty, so the contraction is split in two:
//
//   P[m, (r, q, c)] = sum_t sum_o G_t[m, o] W_t[o, r, q, c]      (m: output pixel)
//   dX[n, h, w, c]  = sum_{r,q} P[(n, i, j), (r, q, c)],  i*s - p + r = h, j*s - p + q = w
//
// The first is a GEMM with output pixels as rows, (r, q, c) as columns
// (KH*KW*C <= 32 * NJB) and K = (t, o).  Each wave takes 32 pixels, loads
// G, T_a and T_b straight from global memory into MFMA fragments (16 bytes
// per lane), forms the products G o T_b and G o T_a once per element, and
// multiplies with weight fragments staged in LDS.  P is fp32 in the
// workspace, tap-major ([r, q][m][c]), so that the second kernel, which
// gathers it over the taps in a fixed order, reads consecutive pixels of one
// tap plane from consecutive lanes.
// Weight fragments of the per-pixel partial sums in LDS: [t][nb][kc][lane],
// lane l: column j = 32 nb + l % 32 of W_t[o, (r, q, c)], output channels
// o = kc KC + VEC (l / 32) .. +VEC (zero past J).
template <typename T, int NJB>
__device__ __forceinline__ void cols_stage_weights(v4u *wfr, const T *__restrict__ w0, const T *__restrict__ w1,
                                                   const T *__restrict__ w2, int O, int J) {
    constexpr int VEC = Elem<T>::VEC;
    constexpr int KC = 2 * VEC;
    const int nkc = O / KC;
    for (int i = threadIdx.x; i < 3 * NJB * nkc * 64; i += blockDim.x) {
        const int l = i & 63, f = i >> 6;
        const int kc = f % nkc, nb = (f / nkc) % NJB, t = f / (nkc * NJB);
        const T *w = t == 0 ? w0 : (t == 1 ? w1 : w2);
        const int j = nb * 32 + (l & 31), o0 = kc * KC + VEC * (l >> 5);
        float v[VEC];
#pragma unroll
        for (int e = 0; e < VEC; ++e) v[e] = j < J ? to_f32<T>(w[(size_t)(o0 + e) * J + j]) : 0.0f;
        wfr[i] = vpack<T>(v);
    }
}

// Partial sums of one wave's 32 output pixels (lane % 32: the pixel whose
// G / T_a / T_b row it loads, m; ok: m is a pixel): acc[nb] holds column
// j = 32 nb + lane % 32 of rows (pixels) 8 (v / 4) + 4 (lane / 32) + v % 4.
template <typename T, int NJB>
__device__ __forceinline__ void cols_group(const T *__restrict__ gy, const T *__restrict__ gta,
                                           const T *__restrict__ gtb, const v4u *wfr, long long m, bool ok, int O,
                                           f32x16_t (&acc)[NJB]) {
    constexpr int VEC = Elem<T>::VEC;
    constexpr int KC = 2 * VEC;  // K elements (output channels) per MFMA chunk
    constexpr int KB = 4;        // chunks whose loads are issued together
    const int lane = threadIdx.x & 63;
    const int nkc = O / KC;
#pragma unroll
    for (int nb = 0; nb < NJB; ++nb)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[nb][v] = 0.0f;
    const size_t rowoff = (size_t)(ok ? m : 0) * O + VEC * (lane >> 5);
    for (int kb = 0; kb < nkc; kb += KB) {
        v4u g[KB], ta[KB], tb[KB];
#pragma unroll
        for (int u = 0; u < KB; ++u) {
            const bool in = ok && kb + u < nkc;
            const size_t off = rowoff + (size_t)(kb + u) * KC;
            g[u] = ld16(gy + off, in);
            ta[u] = ld16(gta + off, in);
            tb[u] = ld16(gtb + off, in);
        }
#pragma unroll
        for (int u = 0; u < KB; ++u) {
            if (kb + u >= nkc) break;
            const int kc = kb + u;
            v4u ga, gb;
            prologue_frag<T>(g[u], ta[u], tb[u], ga, gb);
#pragma unroll
            for (int nb = 0; nb < NJB; ++nb) {
                mfma_chunk<T>(ga, wfr[((0 * NJB + nb) * nkc + kc) * 64 + lane], acc[nb]);
                mfma_chunk<T>(gb, wfr[((1 * NJB + nb) * nkc + kc) * 64 + lane], acc[nb]);
                mfma_chunk<T>(g[u], wfr[((2 * NJB + nb) * nkc + kc) * 64 + lane], acc[nb]);
            }
        }
    }
}

template <typename T, int NJB>
__global__ __launch_bounds__(kThreads) void qconv_bwd_data_cols_kernel(
    const T *__restrict__ gy, const T *__restrict__ gta, const T *__restrict__ gtb, const T *__restrict__ w0,
    const T *__restrict__ w1, const T *__restrict__ w2, float *__restrict__ P, int M, int O, int C, int J) {
    extern __shared__ __attribute__((aligned(16))) v4u wfr[];  // [t][nb][kc][lane]
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    cols_stage_weights<T, NJB>(wfr, w0, w1, w2, O, J);
    __syncthreads();
    // This lane's output column j = 32 nb + lane % 32 is (tap, c) = (j / C, j % C).
    int ptap[NJB], pc[NJB];
#pragma unroll
    for (int nb = 0; nb < NJB; ++nb) {
        const int j = nb * 32 + (lane & 31);
        ptap[nb] = j < J ? j / C : -1;
        pc[nb] = j < J ? j - (j / C) * C : 0;
    }
    const long long nblk = ((long long)M + 31) / 32;
    for (long long mb = (long long)blockIdx.x * (kThreads / 64) + wave; mb < nblk;
         mb += (long long)gridDim.x * (kThreads / 64)) {
        const long long m = mb * 32 + (lane & 31);
        f32x16_t acc[NJB];
        cols_group<T, NJB>(gy, gta, gtb, wfr, m, m < M, O, acc);
        // Lane holds column j = 32 nb + lane % 32 of rows 8 (v / 4) + 4 (lane / 32) + v % 4.
#pragma unroll
        for (int nb = 0; nb < NJB; ++nb) {
            if (ptap[nb] < 0) continue;
            float *plane = P + (size_t)ptap[nb] * M * C + pc[nb];
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const long long row = mb * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
                if (row < M) plane[row * C] = acc[nb][v];
            }
        }
    }
}

// Floats per output pixel of the fused kernel's LDS partial sums: 32 columns
// plus one, so that the gather's threads (consecutive pixels) hit distinct banks.
constexpr int kFusedPitch = 33;

// The two steps above fused for stride 1 (J <= 32): a workgroup takes RB
// input rows h0 .. h0 + RB - 1 of image n.  Their gradient needs the partial
// sums of output rows i = h + PH - r, i.e. i_lo .. i_hi (the band plus a halo
// of KH - 1 rows, recomputed by the neighbouring bands); the waves compute
// those into LDS (one 32-float row per output pixel, column j = (r, q, c)),
// and after one barrier each thread gathers dX[n, h, w, c] over the taps in
// (r, q) order, as the separate gather does.  No partial sums go to HBM.
template <typename T, int NT>
__global__ __launch_bounds__(NT) void qconv_bwd_data_cols_fused_kernel(
    const T *__restrict__ gy, const T *__restrict__ gta, const T *__restrict__ gtb, const T *__restrict__ w0,
    const T *__restrict__ w1, const T *__restrict__ w2, T *__restrict__ dx, int H, int W, int C, int O, int KH,
    int KW, int PH, int PW, int HO, int WO, int RB, int wfr_vecs) {
    extern __shared__ __attribute__((aligned(16))) v4u wfr[];  // weights, then the partial sums
    float *Pl = reinterpret_cast<float *>(wfr + wfr_vecs);     // [local output pixel][kFusedPitch]
    const int J = KH * KW * C;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, lrow = lane & 31;
    const int bands = (H + RB - 1) / RB;
    const int n = blockIdx.x / bands, h0 = (blockIdx.x - n * bands) * RB;
    const int i_lo = max(0, h0 + PH - (KH - 1)), i_hi = min(HO - 1, h0 + RB - 1 + PH);
    const int npx = i_hi >= i_lo ? (i_hi - i_lo + 1) * WO : 0;
    cols_stage_weights<T, 1>(wfr, w0, w1, w2, O, J);
    __syncthreads();
    for (int gl = wave; gl * 32 < npx; gl += NT / 64) {
        const int pl = gl * 32 + lrow;
        const long long m = ((long long)n * HO + i_lo) * WO + pl;  // local pixels are consecutive output pixels
        f32x16_t acc[1];
        cols_group<T, 1>(gy, gta, gtb, wfr, m, pl < npx, O, acc);
        if (lrow < J) {
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int row = gl * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
                if (row < npx) Pl[row * kFusedPitch + lrow] = acc[0][v];
            }
        }
    }
    __syncthreads();
    const int rows = min(RB, H - h0);
    for (int it = threadIdx.x; it < rows * W * C; it += NT) {
        const int hl = it / (W * C), rem = it - hl * (W * C);
        const int w = rem / C, c = rem - w * C;
        const int h = h0 + hl;
        float acc = 0.0f;
        for (int r = 0; r < KH; ++r) {
            const int i = h + PH - r;
            if (i < 0 || i >= HO) continue;
            for (int q = 0; q < KW; ++q) {
                const int j = w + PW - q;
                if (j < 0 || j >= WO) continue;
                acc += Pl[((i - i_lo) * WO + j) * kFusedPitch + (r * KW + q) * C + c];
            }
        }
        dx[(((size_t)n * H + h) * W + w) * C + c] = from_f32<T>(acc);
    }
}

// dX[n, h, w, c] from the tap-major partial sums P ([KH*KW][Mo][C], Mo =
// N*HO*WO): one thread per input pixel, taps summed in (r, q) order.
template <typename T>
__global__ __launch_bounds__(kThreads) void qconv_bwd_data_col2im_kernel(const float *__restrict__ P, T *__restrict__ dx,
                                                                         int N, int H, int W, int C, int KH, int KW,
                                                                         int SH, int SW, int PH, int PW, int HO,
                                                                         int WO) {
    const long long M = (long long)N * H * W;
    const size_t plane = (size_t)N * HO * WO * C;
    for (long long m = (long long)blockIdx.x * blockDim.x + threadIdx.x; m < M;
         m += (long long)gridDim.x * blockDim.x) {
        const int n = (int)(m / ((long long)H * W));
        const int rem = (int)(m - (long long)n * H * W);
        const int h = rem / W, w = rem - (rem / W) * W;
        float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
        for (int r = 0; r < KH; ++r) {
            const int hi = h + PH - r;
            if (hi < 0) break;
            const int i = hi / SH;
            if (i * SH != hi || i >= HO) continue;
            for (int q = 0; q < KW; ++q) {
                const int wi = w + PW - q;
                if (wi < 0) break;
                const int j = wi / SW;
                if (j * SW != wi || j >= WO) continue;
                const float *p = P + (size_t)(r * KW + q) * plane + (((size_t)n * HO + i) * WO + j) * C;
#pragma unroll
                for (int c = 0; c < 4; ++c)
                    if (c < C) acc[c] += p[c];
            }
        }
#pragma unroll
        for (int c = 0; c < 4; ++c)
            if (c < C) dx[m * C + c] = from_f32<T>(acc[c]);
    }
}

// Per-channel statistics of a stored layer output y' (M rows of O channels,
// the forward epilogue's sums when its kernel did not gather them): part p
// takes rows [p rpp, (p + 1) rpp); a thread takes 4 channels of every 16th
// row of the part, and the 16 row lanes are summed in lane order.  Writes
// part[p][0][o] = sum of y', part[p][1][o] = sum of y'^2.
template <typename T>
__global__ __launch_bounds__(kThreads) void qconv_channel_stats_kernel(const T *__restrict__ y, int M, int O,
                                                                        int rpp, float *__restrict__ part) {
    __shared__ float red[2][16][65];
    const int cl = threadIdx.x & 15, rl = threadIdx.x >> 4;
    const int c = blockIdx.y * 64 + 4 * cl;
    const int r0 = blockIdx.x * rpp, r1 = min(M, r0 + rpp);
    float s1[4] = {0.0f, 0.0f, 0.0f, 0.0f}, s2[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    const bool v4 = (O & 3) == 0;
    if (c < O) {
#pragma unroll 4
        for (int r = r0 + rl; r < r1; r += 16) {
            float v[4];
            const T *p = y + (size_t)r * O + c;
            if (v4) {
                load4<T>(p, v);
            } else {
#pragma unroll
                for (int k = 0; k < 4; ++k) v[k] = c + k < O ? to_f32<T>(p[k]) : 0.0f;
            }
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                s1[k] += v[k];
                s2[k] += v[k] * v[k];
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
        if (o < O) part[((size_t)blockIdx.x * 2 + st) * O + o] = t;
    }
}

// Sum of the per-part statistics [part][2][O] in a fixed order: sum[o] and
// sumsq[o].  One workgroup per index j of [2][O] (launch 2 O workgroups).
template <int = 0>  // (a template: defined once across the translation units that include this header)
__global__ __launch_bounds__(kThreads) void qconv_stats_reduce_kernel(const float *__restrict__ part, int nparts,
                                                                       int O, float *sum, float *sumsq) {
    // one sum j per workgroup: thread i adds parts i, i + 256, ... in order, then a fixed tree
    __shared__ float red[kThreads];
    const int j = blockIdx.x, tid = threadIdx.x;
    float s = 0.0f;
#pragma unroll 4
    for (int p = tid; p < nparts; p += kThreads) s += part[(size_t)p * 2 * O + j];
    red[tid] = s;
    __syncthreads();
#pragma unroll
    for (int w = kThreads / 2; w > 0; w >>= 1) {
        if (tid < w) red[tid] += red[tid + w];
        __syncthreads();
    }
    if (tid == 0) {
        if (j < O) sum[j] = red[0];
        else sumsq[j - O] = red[0];
    }
}

}  // namespace ql
