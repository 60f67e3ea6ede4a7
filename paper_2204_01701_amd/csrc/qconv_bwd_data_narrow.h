// qconv_bwd_data_narrow.h -- input gradient of the quadratic convolution
// layer (arXiv 2204.01701, section 4.3, eq:SD) for narrow layers: at most 32
// input channels and a short reduction K = KH * KW * O (the 16-channel stages
// of a CIFAR ResNet), where the tiled kernels spend most of their time on
// per-tile overhead:
//
//   dX[n,h,w,c] = sum_t sum_{o,r,q} W_t[o,r,q,c] G_t[n,(h+p-r)/s,(w+p-q)/s,o]
//   G_a = G o T_b,  G_b = G o T_a,  G_c = G
//
// As in qconv_fwd_narrow.h both MFMA operands arrive in registers straight
// from global memory, in 16-byte runs of the reduction index k = (tap, o):
//   - A (rows = input channels c): the transposed weights W_t^T[c][tap][o],
//     in which a run of o within one tap is contiguous; the three terms'
//     runs are loaded once per wave and stay in registers;
//   - B (columns = input pixels): for input pixel (n, h, w) and tap (r, q)
//     the output pixel ((h + p - r) / s, (w + p - q) / s) when it exists
//     (zero otherwise), whose runs of G, T_a and T_b are contiguous in NHWC;
//     the products G o T_b and G o T_a are formed in fp32 on the run and
//     rounded once to the element type (as in the tiled kernels' prologue);
//   - the 16 x 16 accumulator puts input pixel l % 16 and channels
//     4 (l / 16) .. +4 in lane l: dX of a block is one contiguous run of 16
//     NHWC rows.
// Each wave takes every (waves)-th block of 16 input pixels.
#pragma once

#include "qargs.h"
#include "qdevice.h"
#include "qconv_fwd_narrow.h"

namespace ql {

// CB: 16-channel row blocks (C <= 16 CB, C a multiple of 4).  NCH: reduction
// chunks (K <= NCH narrow_chunk).  S1: stride 1.  O (and so every run) is a
// multiple of the run length.
template <typename T, int CB, int NCH, bool S1>
__global__ __launch_bounds__(kThreads, 2) void qconv_bwd_data_narrow_kernel(const BwdDataArgs a) {
    constexpr int VEC = Elem<T>::VEC;
    constexpr int CK = narrow_chunk<T>();
    const int lane = threadIdx.x & 63, li = lane & 15, lg = lane >> 4;
    const T *__restrict__ gy = static_cast<const T *>(a.gy);
    const T *__restrict__ ta = static_cast<const T *>(a.ta);
    const T *__restrict__ tb = static_cast<const T *>(a.tb);

    // This lane's reduction runs: k = CK ch + VEC lg .. + VEC, tap (r, q), first channel o.
    int kr[NCH], kq[NCH], ko[NCH];
    bool kin[NCH];
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch) {
        const int k = CK * ch + VEC * lg;
        kin[ch] = k < a.K;
        const int tap = (int)fdiv((uint32_t)min(k, a.K - 1), a.fd_o);
        ko[ch] = k - tap * a.O;
        kr[ch] = (int)fdiv((uint32_t)tap, a.fd_kw);
        kq[ch] = tap - kr[ch] * a.KW;
    }
    // The three terms' transposed weight runs: row c = 16 cb + li (zero past C or K).
    v4u wf[3][CB][NCH];
#pragma unroll
    for (int t = 0; t < 3; ++t) {
        const T *__restrict__ wt = static_cast<const T *>(a.wt[t]);
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) {
            const int c = 16 * cb + li;
#pragma unroll
            for (int ch = 0; ch < NCH; ++ch) {
                const int k = CK * ch + VEC * lg;
                wf[t][cb][ch] = (c < a.C && kin[ch]) ? *reinterpret_cast<const v4u *>(wt + (size_t)c * a.K + k)
                                                     : v4u{0u, 0u, 0u, 0u};
            }
        }
    }

    T *__restrict__ dx = static_cast<T *>(a.dx);
    const int nblk = (a.M + 15) / 16;
    const int nw = gridDim.x * (kThreads / 64);
    for (int b = blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6); b < nblk; b += nw) {
        // this lane's input pixel (B column)
        const int p = 16 * b + li;
        const bool pok = p < a.M;
        const int pp = pok ? p : a.M - 1;
        const int n = (int)fdiv((uint32_t)pp, a.fd_hw);
        const int rem = pp - n * a.H * a.W;
        const int h = (int)fdiv((uint32_t)rem, a.fd_w);
        const int w = rem - h * a.W;
        const size_t nbase = (size_t)n * a.HO * a.WO;
        f32x4n_t acc[CB];
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) acc[cb] = f32x4n_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int ch = 0; ch < NCH; ++ch) {
            // the output pixel tap (r, q) of this input pixel reads, if any
            int oh = h + a.PH - kr[ch], ow = w + a.PW - kq[ch];
            bool ok = pok && kin[ch] && oh >= 0 && ow >= 0;
            if constexpr (!S1) {
                const int qh = (int)fdiv((uint32_t)max(oh, 0), a.fd_sh), qw = (int)fdiv((uint32_t)max(ow, 0), a.fd_sw);
                ok = ok && qh * a.SH == oh && qw * a.SW == ow;
                oh = qh;
                ow = qw;
            }
            ok = ok && oh < a.HO && ow < a.WO;
            const size_t off = (nbase + (size_t)oh * a.WO + ow) * a.O + ko[ch];
            const v4u zero = {0u, 0u, 0u, 0u};
            const v4u g = ok ? *reinterpret_cast<const v4u *>(gy + off) : zero;
            const v4u va = ok ? *reinterpret_cast<const v4u *>(ta + off) : zero;
            const v4u vb = ok ? *reinterpret_cast<const v4u *>(tb + off) : zero;
            v4u ga, gb;
            prologue_frag<T>(g, va, vb, ga, gb);
#pragma unroll
            for (int cb = 0; cb < CB; ++cb) {
                narrow_mfma<T>(wf[0][cb][ch], ga, acc[cb]);
                narrow_mfma<T>(wf[1][cb][ch], gb, acc[cb]);
                narrow_mfma<T>(wf[2][cb][ch], g, acc[cb]);
            }
        }
        if (pok) {
#pragma unroll
            for (int cb = 0; cb < CB; ++cb) {
                const int c = 16 * cb + 4 * lg;
                if (c < a.C)
                    store4<T>(dx + (size_t)p * a.C + c, acc[cb][0], acc[cb][1], acc[cb][2], acc[cb][3]);
            }
        }
    }
}

}  // namespace ql
