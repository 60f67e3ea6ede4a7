// qconv_fwd_smallc.h -- forward of the quadratic convolution layer (arXiv
// 2204.01701, section 3.1, eq:2ndneuron3) for layers with few input channels:
// the reduction J = KH * KW * C leaves room for the bias columns below in 32
// (e.g. the RGB stem of an image network, 3 x 3 x 3 = 27).
//
// The whole reduction fits in the k-extent of two bf16 MFMA chunks (four for
// fp32), so there is no K loop, no LDS ring and no zero-padded copy of X:
//   - the three terms' weight fragments (rows o, columns j = (r, q, c), the
//     contiguous OHWI row of W_t) are formed once per workgroup in LDS;
//   - the biases ride in extra reduction columns: pixel value 1, weight value
//     b_t[o], split for bf16 into three bf16 parts whose sum is the fp32 bias
//     exactly (8 + 8 + 8 significand bits), one part for fp32;
//   - each wave takes 32 output pixels at a time and gathers their im2col
//     rows straight from X into pixel fragments (zero outside the image);
//     every lane holds the same 16 columns j for all its pixels, so their
//     (r, q, c) offsets are computed once;
//   - the epilogue forms Y = T_a o T_b + T_c, applies the fused epilogue
//     y' = relu(scale y + shift) when asked, and writes Y, T_a, T_b through a
//     per-wave LDS tile: the 32 pixels are 32 consecutive NHWC rows, so each
//     map's tile is one contiguous run of 32 O elements, copied out in
//     16-byte chunks.  In bf16 the tile holds whole rows (all O channels) of
//     one map, so the chunks cover whole 128-byte cache lines (a 32-channel
//     block alone is half a line); the MFMAs of a map's terms are then redone
//     per map (Y: all three, T_a and T_b: one), a few more cycles of an
//     otherwise idle unit, so that one 32-channel block of accumulators is
//     live.  In fp32 a 32-channel block is a whole line: the tile holds one
//     block of each map in turn, and the three terms' MFMAs run once.
// The layer is bound by the stores of Y, T_a and T_b.
#pragma once

#include "qargs.h"
#include "qdevice.h"

namespace ql {

constexpr int kSmallcK = 32;  // reduction columns of the kernel: J + bias columns

// Bias columns after the J weight columns: three bf16 parts, or one fp32 value.
template <typename T> constexpr int smallc_bias_cols() { return sizeof(T) == 2 ? 3 : 1; }

// Part p of the fp32 bias value b in the element type: bf16 parts are the
// successive round-to-nearest residues (b = p0 + p1 + p2 exactly).
template <typename T> __device__ __forceinline__ float bias_part(float b, int p);
template <> __device__ __forceinline__ float bias_part<float>(float b, int p) { return p == 0 ? b : 0.0f; }
template <> __device__ __forceinline__ float bias_part<uint16_t>(float b, int p) {
    const float p0 = bf2f(f2bf(b));
    const float p1 = bf2f(f2bf(b - p0));
    return p == 0 ? p0 : (p == 1 ? p1 : b - p0 - p1);
}

// OB: 32-row blocks of output channels per term (O = 32 OB), produced one
// at a time (the accumulators of the three terms of one block stay live).
// EPI: apply the fused epilogue (scale, shift, ReLU) to Y.  Each wave takes
// every (gridDim.x * waves)-th group of 32 pixels; the X elements of its next
// group are loaded before the current group's products and stores, so their
// latency overlaps that work.
template <typename T, int OB, bool EPI>
__global__ __launch_bounds__(kThreads, 4) void qconv_fwd_smallc_kernel(const FwdArgs a) {
    constexpr int VEC = Elem<T>::VEC;             // elements per 16-byte fragment
    constexpr int KC = 2 * VEC;                   // reduction columns per MFMA chunk
    constexpr int NKC = kSmallcK / KC;            // chunks covering the 32 columns
    constexpr int NJ = NKC * VEC;                 // columns one lane supplies (16)
    constexpr int NB = smallc_bias_cols<T>();
    constexpr int E = (int)sizeof(T);
    constexpr int O = 32 * OB;
    constexpr bool ROWS = E == 2;                 // bf16: whole rows of one map per tile
    constexpr int SB = ROWS ? O : 32;             // channels of a staged pixel row
    constexpr int PITCH = SB * E + 16;            // LDS bytes per staged pixel row
    constexpr int CPR = SB * E / 16;              // 16-byte chunks per staged row
    constexpr int NWAVE = kThreads / 64;
    constexpr int NWF = 3 * OB * NKC;             // weight fragments
    __shared__ __attribute__((aligned(16))) v4u wfr[NWF][64];
    __shared__ __attribute__((aligned(16))) char stage[NWAVE][32 * PITCH];

    const int tid = threadIdx.x, lane = tid & 63, lrow = lane & 31, lhi = lane >> 5, wave = tid >> 6;
    const int J = a.K;
    char *buf = stage[wave];

    // Weight fragments (term t, row block ob, chunk kc; row o = 32 ob + l % 32,
    // column j = kc KC + VEC (l / 32) + e), bias parts in columns J .. J + NB - 1.
    for (int i = tid; i < NWF * 64; i += kThreads) {
        const int l = i & 63, f = i >> 6;
        const int kc = f % NKC, ob = (f / NKC) % OB, t = f / (NKC * OB);
        const int o = 32 * ob + (l & 31);
        const T *__restrict__ w = static_cast<const T *>(a.w[t]);
        const float b = a.bias[t] ? a.bias[t][o] : 0.0f;
        float v[VEC];
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
            const int j = kc * KC + VEC * (l >> 5) + e;
            v[e] = j < J ? to_f32<T>(w[(size_t)o * J + j]) : (j < J + NB ? bias_part<T>(b, j - J) : 0.0f);
        }
        wfr[f][l] = vpack<T>(v);
    }
    // Column table of each lane half h: element i -> j = (i / VEC) KC + VEC h + i % VEC,
    // {element offset of (r, q, c) in X, (r << 16) | q}, or {0, -1} past J.
    __shared__ int2 jtab[2][NJ];
    if (tid < 2 * NJ) {
        const int h = tid / NJ, i = tid % NJ;
        const int j = (i / VEC) * KC + VEC * h + (i % VEC);
        const int tap = (int)fdiv((uint32_t)j, a.fd_c), c = j - tap * a.C;
        const int r = (int)fdiv((uint32_t)tap, a.fd_kw), q = tap - r * a.KW;
        jtab[h][i] = j < J ? make_int2((r * a.W + q) * a.C + c, (r << 16) | q) : make_int2(0, -1);
    }
    // bias columns of this lane (value 1); columns past J + NB stay zero
    uint32_t ones = 0;
#pragma unroll
    for (int i = 0; i < NJ; ++i) {
        const int j = (i / VEC) * KC + VEC * lhi + (i % VEC);
        if (j >= J && j < J + NB) ones |= 1u << i;
    }
    __syncthreads();

    const T *__restrict__ x = static_cast<const T *>(a.x);
    T *outs[3] = {static_cast<T *>(a.y), static_cast<T *>(a.ta), static_cast<T *>(a.tb)};
    const long long ngroups = ((long long)a.M + 31) / 32;
    const long long stride = (long long)gridDim.x * NWAVE;
    // X elements of group g for this lane's pixel: unconditional loads (a
    // column outside the image reads element 0), the in-bounds bits in `inb`.
    T raw[NJ];
    uint32_t inb = 0;
    auto gather = [&](long long g) {
        const long long m = g * 32 + lrow;
        const bool mok = m < a.M;
        const int mm = mok ? (int)m : 0;
        const int n = (int)fdiv((uint32_t)mm, a.fd_howo);
        const int rem = mm - n * a.HO * a.WO;
        const int oh = (int)fdiv((uint32_t)rem, a.fd_wo);
        const int ow = rem - oh * a.WO;
        const int h0 = oh * a.SH - a.PH, w0 = ow * a.SW - a.PW;
        const long long base = ((long long)(n * a.H + h0) * a.W + w0) * a.C;
        inb = 0;
#pragma unroll
        for (int i = 0; i < NJ; ++i) {
            const int2 jt = jtab[lhi][i];
            const int rq = jt.y;
            const bool in = rq >= 0 && mok && (unsigned)(h0 + (rq >> 16)) < (unsigned)a.H &&
                            (unsigned)(w0 + (rq & 0xffff)) < (unsigned)a.W;
            raw[i] = x[in ? base + jt.x : 0];
            inb |= (uint32_t)in << i;
        }
    };
    long long gi = (long long)blockIdx.x * NWAVE + wave;
    if (gi < ngroups) gather(gi);
    for (; gi < ngroups; gi += stride) {
        // this group's pixel fragments, then the next group's loads
        v4u pf[NKC];
        {
            float v[NJ];
#pragma unroll
            for (int i = 0; i < NJ; ++i)
                v[i] = ((inb >> i) & 1u) ? to_f32<T>(raw[i]) : (((ones >> i) & 1u) ? 1.0f : 0.0f);
#pragma unroll
            for (int kc = 0; kc < NKC; ++kc) pf[kc] = vpack<T>(v + kc * VEC);
        }
        const long long m0 = gi * 32;
        if (gi + stride < ngroups) gather(gi + stride);
        // Map jm = 0: Y (through the fused epilogue), 1: T_a, 2: T_b.
        // terms(): the accumulators of 32-channel block ob (only term jm - 1
        // for map jm > 0 when `need` is set); emit(): block ob of map jm into
        // channels 32 slot .. +32 of the staged rows; flush(): the staged
        // rows of map jm to channels c0 .. c0 + SB of its 32 NHWC rows.
        f32x16_t acc[3];
        auto terms = [&](int ob, int jm, bool need) {
#pragma unroll
            for (int t = 0; t < 3; ++t) {
                if (need && jm != 0 && t != jm - 1) continue;
#pragma unroll
                for (int v = 0; v < 16; ++v) acc[t][v] = 0.0f;
#pragma unroll
                for (int kc = 0; kc < NKC; ++kc) mfma_chunk<T>(wfr[(t * OB + ob) * NKC + kc][lane], pf[kc], acc[t]);
            }
        };
        auto emit = [&](int jm, int ob, int slot) {
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int ol = 8 * g + 4 * lhi;
                float v[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int k = 4 * g + i;
                    v[i] = jm == 1 ? acc[0][k] : (jm == 2 ? acc[1][k] : acc[0][k] * acc[1][k] + acc[2][k]);
                    if constexpr (EPI) {
                        if (jm == 0) v[i] = epi_apply(a.epi, 32 * ob + ol + i, v[i]);
                    }
                }
                store4<T>(reinterpret_cast<T *>(buf + lrow * PITCH + (32 * slot + ol) * E), v[0], v[1], v[2], v[3]);
            }
        };
        auto flush = [&](int jm, int c0) {
            wave_lds_sync();
            T *__restrict__ dst = outs[jm] + m0 * O + c0;
#pragma unroll
            for (int c = lane; c < 32 * CPR; c += 64) {
                const int row = c / CPR, cc = c - (c / CPR) * CPR;
                if (m0 + row < a.M)
                    *reinterpret_cast<v4u *>(dst + (size_t)row * O + cc * (16 / E)) = lds_read16(buf + row * PITCH + cc * 16);
            }
            wave_lds_sync();  // the tile is read before the next map overwrites it
        };
        if constexpr (ROWS) {
#pragma unroll
            for (int jm = 0; jm < 3; ++jm) {
                if (!outs[jm]) continue;
#pragma unroll
                for (int ob = 0; ob < OB; ++ob) {
                    terms(ob, jm, true);
                    emit(jm, ob, ob);
                }
                flush(jm, 0);
            }
        } else {
#pragma unroll
            for (int ob = 0; ob < OB; ++ob) {
                terms(ob, 0, false);
#pragma unroll
                for (int jm = 0; jm < 3; ++jm) {
                    if (!outs[jm]) continue;
                    emit(jm, ob, 0);
                    flush(jm, 32 * ob);
                }
            }
        }
    }
}

}  // namespace ql
