// qconv_bwd_weight_narrow.h -- weight and bias gradients of the quadratic
// convolution layer (arXiv 2204.01701, section 4.3, eq:SD) for narrow layers:
// at most 16 output channels and a short row k' = (r, q, c) (KH KW C <= 144,
// the 16-channel stages of a CIFAR ResNet and its 3-channel stem, X zero-padded
// to whole 16-byte runs), where the tiled kernels'
// 64-channel, 128-row tiles leave most of their MFMA work on zero padding:
//
//   dW_t[o,r,q,c] = sum_{n,i,j} G_t[n,i,j,o] X[n, i*s-p+r, j*s-p+q, c]
//   db_t[o]       = sum_{n,i,j} G_t[n,i,j,o]
//   G_a = G o T_b,  G_b = G o T_a,  G_c = G
//
// The tile is the whole gradient: all k' rows (NF fragments of 16) by the 16
// output channels of all three terms, so every MFMA is useful work (wider
// layers, up to 64 channels such as the 3-channel stem of a CIFAR VGG-16,
// take one 16-channel slice per workgroup row of the grid).  Each
// wave runs its own contiguous range of K steps (KE output pixels) with a
// private LDS area and no barriers:
//   - its lanes load the step's im2col rows of X (one 16-byte run of k' per
//     lane and fragment, lane = (pixel, run group)) and the runs of G, T_a,
//     T_b, form the products G o T_b, G o T_a in fp32 (the bias sums add
//     them before rounding) and write all of it to LDS as pixel rows, the
//     next step's loads already in flight where the registers allow;
//   - the MFMA operands come back transposed (pixels as the reduction index):
//     bf16 by ds_read_b64_tr_b16 into v_mfma_f32_16x16x32_bf16, fp32 by
//     ds_read_b32 into v_mfma_f32_16x16x4f32 (rows padded by 16 bytes, so
//     both the row writes and the transposing reads are free of bank
//     conflicts).
// The four waves' sums are added in LDS in wave order; the workgroup writes
// its part (or, as the only split, dW_t and db_t themselves).
#pragma once

#include "qargs.h"
#include "qdevice.h"
#include "qpipe.h"

namespace ql {

typedef float f32x4w_t __attribute__((ext_vector_type(4)));

// bf16 operand (16 GEMM rows x 32 pixels) from an LDS tile of pixel rows
// (pitch bytes each; GEMM column m contiguous): lane l gets GEMM row m0 + l % 16
// and pixels 8 (l / 16) .. +8.  In a group g of 16 lanes, lane j addresses
// pixel row 8 g + 4 h + j / 4, columns m0 + 4 (j % 4) .. +4, so that the
// transposing read hands lane i column m0 + i of four consecutive pixels.
__device__ __forceinline__ v4u narrow_tr_frag(const char *tile, int pitch, int m0, int lane) {
    const int g = lane >> 4, j = lane & 15;
    const int col = m0 + 4 * (j & 3);
    v4u out;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int row = 8 * g + 4 * h + (j >> 2);
        const v4s_t v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s_t *)(tile + row * pitch + col * 2));
        const v2u w = __builtin_bit_cast(v2u, v);
        out[2 * h] = w.x;
        out[2 * h + 1] = w.y;
    }
    return out;
}

// NF: 16-row k' fragments (KP <= 16 NF).  SUM: the bias sums too.
template <typename T, int NF, bool SUM>
__device__ __forceinline__ void bwd_weight_narrow_body(const BwdWeightArgs &a, char *smem) {
    constexpr bool BF = sizeof(T) == 2;
    constexpr int VEC = Elem<T>::VEC;  // elements per 16-byte run
    constexpr int KE = BF ? 32 : 16;   // output pixels per K step (one MFMA reduction extent, four for fp32)
    constexpr int RG = 64 / KE;        // lanes per pixel: the runs of 16 k' (or 16 channels)
    constexpr int RUNS = RG * NF;      // runs per X row
    constexpr int XP = 16 * RUNS + 16, PP = 16 * RG + 16;  // row pitches (bytes)
    constexpr int XT = KE * XP, PT = KE * PP;
    constexpr int WAVE_LDS = XT + 3 * PT;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    char *const xt = smem + wave * WAVE_LDS;
    char *const pt = xt + XT;
    const int px = lane % KE, rg = lane / KE;
    const T *__restrict__ x = static_cast<const T *>(a.x);
    const T *__restrict__ gsrc[3] = {static_cast<const T *>(a.gy), static_cast<const T *>(a.ta),
                                     static_cast<const T *>(a.tb)};

    // this lane's X runs: fragment i, k' = 16 i + VEC rg .. + VEC (one tap)
    int xr[NF], xq[NF], xc[NF];
    bool kok[NF];
#pragma unroll
    for (int i = 0; i < NF; ++i) {
        const int k = 16 * i + VEC * rg;
        kok[i] = k < a.KP;
        const int tap = (int)fdiv((uint32_t)min(k, a.KP - 1), a.fd_c);
        xc[i] = k - tap * a.C;
        xr[i] = (int)fdiv((uint32_t)tap, a.fd_kw);
        xq[i] = tap - xr[i] * a.KW;
    }
    // this workgroup's 16 output channels ob0 .. ob0 + 16 (blockIdx.y), and
    // this lane's G-side run of them: channels ob0 + o0 .. + VEC
    const int ob0 = blockIdx.y * 16;
    const int o0 = VEC * rg;
    const bool ook = ob0 + o0 < a.O;

    // this wave's K steps: a contiguous quarter of the workgroup's
    const int split = blockIdx.x;
    const int w_begin = split * a.stages_per_split;
    const int w_end = min(a.stages_total, w_begin + a.stages_per_split);
    const int q = (w_end - w_begin + 3) / 4;
    const int s_begin = min(w_end, w_begin + wave * q), s_end = min(w_end, s_begin + q);

    auto load = [&](int s, v4u *xv, v4u *gv) {
        const int m = s * KE + px;
        const bool mok = s < s_end && m < a.M;
        const int mm = mok ? m : 0;
        const int n = (int)fdiv((uint32_t)mm, a.fd_howo);
        const int rem = mm - n * a.HO * a.WO;
        const int oh = (int)fdiv((uint32_t)rem, a.fd_wo);
        const int ow = rem - oh * a.WO;
        const int h0 = oh * a.SH - a.PH, w0 = ow * a.SW - a.PW;
        const v4u zero = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int i = 0; i < NF; ++i) {
            const int ih = h0 + xr[i], iw = w0 + xq[i];
            const bool ok = mok && kok[i] && (unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W;
            xv[i] = ok ? *reinterpret_cast<const v4u *>(x + ((size_t)(n * a.H + ih) * a.W + iw) * a.C + xc[i]) : zero;
        }
        const bool gok = mok && ook;
        const size_t off = (size_t)mm * a.O + ob0 + o0;
#pragma unroll
        for (int u = 0; u < 3; ++u) gv[u] = gok ? *reinterpret_cast<const v4u *>(gsrc[u] + off) : zero;
    };

    f32x4w_t acc[3][NF];
#pragma unroll
    for (int t = 0; t < 3; ++t)
#pragma unroll
        for (int i = 0; i < NF; ++i) acc[t][i] = f32x4w_t{0.0f, 0.0f, 0.0f, 0.0f};
    float dsum[3][VEC];
#pragma unroll
    for (int t = 0; t < 3; ++t)
#pragma unroll
        for (int e = 0; e < VEC; ++e) dsum[t][e] = 0.0f;

    constexpr bool PF = NF <= 6;  // load the next step during this one (longer rows: its registers would spill)
    v4u xv[NF], gv[3];
    if constexpr (PF) load(s_begin, xv, gv);
    for (int s = s_begin; s < s_end; ++s) {
        if constexpr (!PF) load(s, xv, gv);
        // the step's rows into LDS: X runs, then G o T_b, G o T_a, G
        float fa[VEC], fb[VEC];
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
            const float gval = vget<T>(gv[0], e);
            fa[e] = gval * vget<T>(gv[2], e);
            fb[e] = gval * vget<T>(gv[1], e);
            if constexpr (SUM) {
                dsum[0][e] += fa[e];
                dsum[1][e] += fb[e];
                dsum[2][e] += gval;
            }
        }
#pragma unroll
        for (int i = 0; i < NF; ++i) *reinterpret_cast<v4u *>(xt + px * XP + (rg + RG * i) * 16) = xv[i];
        *reinterpret_cast<v4u *>(pt + px * PP + rg * 16) = vpack<T>(fa);
        *reinterpret_cast<v4u *>(pt + PT + px * PP + rg * 16) = vpack<T>(fb);
        *reinterpret_cast<v4u *>(pt + 2 * PT + px * PP + rg * 16) = gv[0];
        if constexpr (PF) {
            if (s + 1 < s_end) load(s + 1, xv, gv);  // (registers free once written)
        }
        wave_lds_sync();
        if constexpr (BF) {
            v4u bt[3];
#pragma unroll
            for (int t = 0; t < 3; ++t) bt[t] = narrow_tr_frag(pt + t * PT, PP, 0, lane);
#pragma unroll
            for (int i = 0; i < NF; ++i) {
                const v4u af = narrow_tr_frag(xt, XP, 16 * i, lane);
#pragma unroll
                for (int t = 0; t < 3; ++t)
                    acc[t][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, af),
                                                                        __builtin_bit_cast(bf16x8_t, bt[t]),
                                                                        acc[t][i], 0, 0, 0);
            }
        } else {
            // four reduction chunks of 4 pixels: lane l reads pixel 4 c + l / 16, column l % 16
            const int pr = lane >> 4, col = lane & 15;
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                float bt[3];
#pragma unroll
                for (int t = 0; t < 3; ++t)
                    bt[t] = *reinterpret_cast<const float *>(pt + t * PT + (4 * c + pr) * PP + col * 4);
#pragma unroll
                for (int i = 0; i < NF; ++i) {
                    const float af = *reinterpret_cast<const float *>(xt + (4 * c + pr) * XP + (16 * i + col) * 4);
#pragma unroll
                    for (int t = 0; t < 3; ++t)
                        acc[t][i] = __builtin_amdgcn_mfma_f32_16x16x4f32(af, bt[t], acc[t][i], 0, 0, 0);
                }
            }
        }
        wave_lds_sync();  // the reads are done before the next step's rows overwrite them
    }

    // The four waves' sums, term by term, in wave order (wave 0 keeps the total).
    // Lane l holds channel o = l % 16, rows k' = 16 i + 4 (l / 16) .. +4.
    float *red = reinterpret_cast<float *>(smem);
    static_assert((3 * NF * 4 * 64 + 4 * 3 * 16) * 4 <= 4 * WAVE_LDS, "reduction area fits");
#pragma unroll
    for (int t = 0; t < 3; ++t) {
        __syncthreads();
        if (wave > 0) {
#pragma unroll
            for (int i = 0; i < NF; ++i)
#pragma unroll
                for (int v = 0; v < 4; ++v) red[(((wave - 1) * NF + i) * 4 + v) * 64 + lane] = acc[t][i][v];
        }
        __syncthreads();
        if (wave == 0) {
#pragma unroll
            for (int w = 0; w < 3; ++w)
#pragma unroll
                for (int i = 0; i < NF; ++i)
#pragma unroll
                    for (int v = 0; v < 4; ++v) acc[t][i][v] += red[((w * NF + i) * 4 + v) * 64 + lane];
        }
    }
    // bias sums: the KE lanes of a run group add in a fixed butterfly, then the waves in order
    float *dred = red + 3 * NF * 4 * 64;  // [wave][3][16]
    if constexpr (SUM) {
#pragma unroll
        for (int t = 0; t < 3; ++t)
#pragma unroll
            for (int e = 0; e < VEC; ++e) {
                float v = dsum[t][e];
#pragma unroll
                for (int d = 1; d < KE; d <<= 1) v += __shfl_xor(v, d);
                dsum[t][e] = v;
            }
        __syncthreads();
        if (px == 0) {
#pragma unroll
            for (int t = 0; t < 3; ++t)
#pragma unroll
                for (int e = 0; e < VEC; ++e) dred[(wave * 3 + t) * 16 + o0 + e] = dsum[t][e];
        }
        __syncthreads();
    }
    if (wave != 0) return;
    const int ol = lane & 15, o = ob0 + ol, lg = lane >> 4;
    // dW_t rows as stored: KH KW C_out (X zero-padded to C channels: the padded columns are dropped)
    const bool padded = a.C_out != a.C;
    const int KPO = a.KH * a.KW * a.C_out;
#pragma unroll
    for (int t = 0; t < 3; ++t) {
        float *__restrict__ dst = a.splits == 1 ? a.dw[t] : a.ws_dw + ((size_t)split * 3 + t) * (size_t)a.O * KPO;
        if (o < a.O) {
#pragma unroll
            for (int i = 0; i < NF; ++i) {
                const int k = 16 * i + 4 * lg;
                if (k >= a.KP) continue;
                if (!padded) {
                    *reinterpret_cast<v4f *>(dst + (size_t)o * a.KP + k) =
                        v4f{acc[t][i][0], acc[t][i][1], acc[t][i][2], acc[t][i][3]};
                } else {
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        const int tap = (int)fdiv((uint32_t)(k + v), a.fd_c);
                        const int c = k + v - tap * a.C;
                        if (c < a.C_out) dst[(size_t)o * KPO + tap * a.C_out + c] = acc[t][i][v];
                    }
                }
            }
        }
        if constexpr (SUM) {
            if (lg == 0 && o < a.O) {
                const float tot = dred[(0 * 3 + t) * 16 + ol] + dred[(1 * 3 + t) * 16 + ol] +
                                  dred[(2 * 3 + t) * 16 + ol] + dred[(3 * 3 + t) * 16 + ol];
                if (a.splits == 1) a.db[t][o] = tot;
                else a.ws_db[((size_t)split * 3 + t) * a.O + o] = tot;
            }
        }
    }
}

template <typename T, int NF>
__global__ __launch_bounds__(kThreads, 2) void qconv_bwd_weight_narrow_kernel(const BwdWeightArgs a) {
    constexpr int KE = sizeof(T) == 2 ? 32 : 16, RG = 64 / KE;
    constexpr int WAVE_LDS = KE * (16 * RG * NF + 16) + 3 * KE * (16 * RG + 16);
    __shared__ __attribute__((aligned(16))) char smem[4 * WAVE_LDS];
    if (a.want_db) bwd_weight_narrow_body<T, NF, true>(a, smem);
    else bwd_weight_narrow_body<T, NF, false>(a, smem);
}

}  // namespace ql
