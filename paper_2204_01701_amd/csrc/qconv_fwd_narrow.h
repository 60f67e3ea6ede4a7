// qconv_fwd_narrow.h -- forward of the quadratic convolution layer (arXiv
// 2204.01701, section 3.1, eq:2ndneuron3) for narrow layers: at most 32 output
// channels and a short reduction J = KH * KW * C (the 16-channel stages of a
// CIFAR ResNet and its stem), where the tiled implicit GEMM spends most of
// its time on per-tile overhead (three 64-row term blocks for 16 channels).
//
// Both MFMA operands arrive in registers in their fragment layout straight
// from global memory, with no LDS:
//   - the 16 x 16 MFMA operand of a lane is one 16-byte run of the reduction
//     index (8 bf16 or 4 fp32 values); with channels-last X and OHWI weights
//     a run of j = (r, q, c) within one tap is contiguous in both, so a lane
//     of column (pixel) l % 16 loads its run of X with one 16-byte load, and
//     a lane of row (output channel) l % 16 its run of W_t;
//   - the three terms' weight fragments (rows o, all of J) are loaded once per
//     wave and stay in registers; each wave then takes every (waves)-th block
//     of 16 output pixels, loading the next block's X runs before the current
//     block's MFMAs where the registers allow (J of at most 6 runs per lane);
//   - the 16 x 16 accumulator layout puts pixel l % 16 and channels
//     4 (l / 16) .. +4 in lane l, so the epilogue forms Y = T_a o T_b + T_c
//     (with the fused scale, shift, ReLU when asked) in place and each map of
//     a block is one contiguous run of 16 NHWC rows.
// With the statistics of the forward epilogue requested, each lane sums the
// stored Y' of its four channels over the wave's blocks; the 16 lanes of a
// channel group add theirs in a fixed butterfly and the wave writes one part
// (sum, then sum of squares, per channel), reduced later in part order.
// fp32 uses v_mfma_f32_16x16x4f32: a lane's 16-byte run (4 values) feeds four
// MFMAs, value i to the i-th, the weight runs split the same way, so the
// four MFMAs together cover the run's reduction indices once.
#pragma once

#include "qargs.h"
#include "qdevice.h"

namespace ql {

typedef float f32x4n_t __attribute__((ext_vector_type(4)));

// acc(16 x 16) += A(16 rows x run) * B(run x 16 columns) over one 16-byte run
// per lane: bf16 one v_mfma_f32_16x16x32_bf16, fp32 four v_mfma_f32_16x16x4f32.
template <typename T> __device__ __forceinline__ void narrow_mfma(const v4u &a, const v4u &b, f32x4n_t &acc);
template <> __device__ __forceinline__ void narrow_mfma<uint16_t>(const v4u &a, const v4u &b, f32x4n_t &acc) {
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                  acc, 0, 0, 0);
}
template <> __device__ __forceinline__ void narrow_mfma<float>(const v4u &a, const v4u &b, f32x4n_t &acc) {
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
}

// Reduction elements one 16-byte run per lane covers across the four lane
// groups of a 16 x 16 operand: 32 bf16 or 16 fp32.
template <typename T> constexpr int narrow_chunk() { return 4 * Elem<T>::VEC; }

// OB: 16-channel row blocks per term (O <= 16 OB, O a multiple of 4).  NCH:
// reduction chunks (J <= NCH narrow_chunk).  EPI: the fused epilogue on Y.
// C (the channels the kernel sees) is a multiple of the run length, so no
// run crosses a tap.
template <typename T, int OB, int NCH, bool EPI>
__global__ __launch_bounds__(kThreads, 2) void qconv_fwd_narrow_kernel(const FwdArgs a) {
    constexpr int VEC = Elem<T>::VEC;
    constexpr int CK = narrow_chunk<T>();
    const int lane = threadIdx.x & 63, li = lane & 15, lg = lane >> 4;
    const T *__restrict__ x = static_cast<const T *>(a.x);

    // This lane's reduction runs: k = CK ch + VEC lg .. + VEC, tap (r, q), channel c.
    int kdr[NCH], kdq[NCH], kc[NCH];
    bool kin[NCH];
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch) {
        const int k = CK * ch + VEC * lg;
        kin[ch] = k < a.K;
        const int tap = (int)fdiv((uint32_t)min(k, a.K - 1), a.fd_c);
        kc[ch] = k - tap * a.C;
        const int r = (int)fdiv((uint32_t)tap, a.fd_kw);
        kdr[ch] = r - a.PH;
        kdq[ch] = tap - r * a.KW - a.PW;
    }
    // The three terms' weight runs: row o = 16 ob + li (zero past O or J).
    v4u wf[3][OB][NCH];
#pragma unroll
    for (int t = 0; t < 3; ++t) {
        const T *__restrict__ w = static_cast<const T *>(a.w[t]);
#pragma unroll
        for (int ob = 0; ob < OB; ++ob) {
            const int o = 16 * ob + li;
#pragma unroll
            for (int ch = 0; ch < NCH; ++ch) {
                const int k = CK * ch + VEC * lg;
                wf[t][ob][ch] = (o < a.O && kin[ch]) ? *reinterpret_cast<const v4u *>(w + (size_t)o * a.K + k)
                                                     : v4u{0u, 0u, 0u, 0u};
            }
        }
    }
    // Accumulator rows of this lane: o = 16 ob + 4 lg + v; their biases.
    float bias[3][OB][4];
#pragma unroll
    for (int t = 0; t < 3; ++t)
#pragma unroll
        for (int ob = 0; ob < OB; ++ob)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int o = 16 * ob + 4 * lg + v;
                bias[t][ob][v] = (a.bias[t] != nullptr && o < a.O) ? a.bias[t][o] : 0.0f;
            }

    // X runs of the block's pixel m = 16 b + li (zero outside the image or past J or M).
    auto load_x = [&](int b, v4u *xf) {
        const int m = 16 * b + li;
        const bool mok = m < a.M;
        const int mm = mok ? m : a.M - 1;
        const int n = (int)fdiv((uint32_t)mm, a.fd_howo);
        const int rem = mm - n * a.HO * a.WO;
        const int oh = (int)fdiv((uint32_t)rem, a.fd_wo);
        const int ow = rem - oh * a.WO;
        const int h0 = oh * a.SH, w0 = ow * a.SW;
        const size_t nbase = (size_t)n * a.H * a.W;
#pragma unroll
        for (int ch = 0; ch < NCH; ++ch) {
            const int ih = h0 + kdr[ch], iw = w0 + kdq[ch];
            const bool ok = mok && kin[ch] && (unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W;
            xf[ch] = ok ? *reinterpret_cast<const v4u *>(x + (nbase + (size_t)ih * a.W + iw) * a.C + kc[ch])
                        : v4u{0u, 0u, 0u, 0u};
        }
    };

    T *__restrict__ y = static_cast<T *>(a.y);
    T *__restrict__ ta = static_cast<T *>(a.ta);
    T *__restrict__ tb = static_cast<T *>(a.tb);
    const int nblk = (a.M + 15) / 16;
    const int nw = gridDim.x * (kThreads / 64);
    const int wid = blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
    int b = wid;
    const bool stats = EPI && a.stat_part != nullptr;
    float ssum[OB][4], ssq[OB][4];
#pragma unroll
    for (int ob = 0; ob < OB; ++ob)
#pragma unroll
        for (int v = 0; v < 4; ++v) ssum[ob][v] = ssq[ob][v] = 0.0f;
    constexpr bool PF = NCH <= 6;  // prefetch the next block (longer J: its registers would spill)
    v4u xf[NCH];
    if constexpr (PF) load_x(b, xf);
    for (; b < nblk; b += nw) {
        v4u xn[PF ? NCH : 1];
        if constexpr (PF) {
            if (b + nw < nblk) load_x(b + nw, xn);
        } else {
            load_x(b, xf);
        }
        f32x4n_t acc[3][OB];
#pragma unroll
        for (int t = 0; t < 3; ++t)
#pragma unroll
            for (int ob = 0; ob < OB; ++ob)
                acc[t][ob] = f32x4n_t{bias[t][ob][0], bias[t][ob][1], bias[t][ob][2], bias[t][ob][3]};
#pragma unroll
        for (int ch = 0; ch < NCH; ++ch)
#pragma unroll
            for (int t = 0; t < 3; ++t)
#pragma unroll
                for (int ob = 0; ob < OB; ++ob) narrow_mfma<T>(wf[t][ob][ch], xf[ch], acc[t][ob]);
        const int m = 16 * b + li;
        if (m < a.M) {
#pragma unroll
            for (int ob = 0; ob < OB; ++ob) {
                const int o = 16 * ob + 4 * lg;
                if (o >= a.O) continue;
                const size_t off = (size_t)m * a.O + o;
                float yv[4];
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    yv[v] = acc[0][ob][v] * acc[1][ob][v] + acc[2][ob][v];
                    if constexpr (EPI) yv[v] = epi_apply(a.epi, o + v, yv[v]);
                }
                if (y) store4<T>(y + off, yv[0], yv[1], yv[2], yv[3]);
                if (stats) {
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        const float f = to_f32<T>(from_f32<T>(yv[v]));  // the stored value
                        ssum[ob][v] += f;
                        ssq[ob][v] += f * f;
                    }
                }
                if (ta) store4<T>(ta + off, acc[0][ob][0], acc[0][ob][1], acc[0][ob][2], acc[0][ob][3]);
                if (tb) store4<T>(tb + off, acc[1][ob][0], acc[1][ob][1], acc[1][ob][2], acc[1][ob][3]);
            }
        }
        if constexpr (PF) {
#pragma unroll
            for (int ch = 0; ch < NCH; ++ch) xf[ch] = xn[ch];
        }
    }
    if (stats) {
        // this wave's part: the 16 lanes of channel group lg add in a fixed butterfly
        float *part = a.stat_part + (size_t)wid * 2 * a.O;
#pragma unroll
        for (int ob = 0; ob < OB; ++ob)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                float s1 = ssum[ob][v], s2 = ssq[ob][v];
#pragma unroll
                for (int d = 1; d < 16; d <<= 1) {
                    s1 += __shfl_xor(s1, d);
                    s2 += __shfl_xor(s2, d);
                }
                const int o = 16 * ob + 4 * lg + v;
                if (li == 0 && o < a.O) {
                    part[o] = s1;
                    part[a.O + o] = s2;
                }
            }
    }
}

}  // namespace ql
