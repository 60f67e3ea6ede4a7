// qconv_bwd_weight16.h -- weight and bias gradients of the quadratic
// convolution layer (arXiv 2204.01701, section 4.3, eq:SD), the pipelined
// bf16 kernel with 16 x 16 x 32 MFMA tiles:
//
//   dW_t[o,r,q,c] = sum_{n,i,j} G_t[n,i,j,o] X[n, i*s-p+r, j*s-p+q, c]
//   db_t[o]       = sum_{n,i,j} G_t[n,i,j,o]
//   G_a = G o T_b,  G_b = G o T_a,  G_c = G
//
// The same implicit GEMM and LDS ring as qconv_bwd_weight.h (rows k' =
// (r, q, c), columns (t, o), K = output pixels, split-K), but the four waves
// of a workgroup sit side by side over the output channels, each covering
// every k' row of the tile for 16 channels of all three terms.  The G-side
// operands of a wave (16 channels x 32 pixels of G, T_a, T_b) then feed the
// MFMAs of all eight 16-row k' fragments, and no two waves form the same
// products: each product G o T_b, G o T_a is formed once per workgroup, where
// the 2 x 2 wave grid of the 32 x 32 kernel forms it twice.  With the
// 16 x 16 x 32 instruction the 128 x 16 x 3 wave tile takes 96 accumulator
// registers (a 128 x 32 x 3 tile of 32 x 32 MFMAs would take 192), so two
// workgroups still share a CU.
//
// A K step is one 32-pixel MFMA k-chunk.  The ring's two register sets hold
// the step's k' fragments 0-3 (set 0, with the G-side fragments) and 4-7
// (set 1); the products are formed once per step, in the first half.
//
// BO = 128 puts eight waves side by side (one workgroup per CU, 160 KB of
// LDS): each K step copies 32 KB for twice the MFMAs of a 64-channel tile's
// 20 KB, so the same LDS holds more MFMA work in flight.
//
// KG = 2 runs two such 4-wave pipelines in one 8-wave workgroup (one per CU,
// each pipeline with its own LDS ring), on the two halves of the
// workgroup's K range, and adds their accumulators in LDS before the
// epilogue: half the workgroups, and so half the fp32 split-K partial sums
// (written and read back once each), of two 4-wave workgroups per CU, at the
// same occupancy.  The sum of the two halves is taken in a fixed order, so
// the result stays bitwise repeatable.
#pragma once

#include "qargs.h"
#include "qpipe.h"

namespace ql {

typedef float f32x4_t __attribute__((ext_vector_type(4)));

// acc(16x16) += A(16 x 32) * B(32 x 16), bf16 operands: lane l holds row (A)
// or column (B) l % 16 and reduction values 8 (l / 16) .. +8; the result
// lane l holds column l % 16, rows 4 (l / 16) .. +4.
__device__ __forceinline__ void mfma16(const v4u &a, const v4u &b, f32x4_t &acc) {
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                  acc, 0, 0, 0);
}

// LDS tiles of this kernel: the NAT layout of qpipe.h (rows = reduction
// index, 16-byte slots of GEMM columns) with a swizzle of its own.  One
// fragment read below covers, per half-wave, the rows 8 g + 4 h + 0..3 of two
// lane groups g (8 rows apart) at the same two slots; the swizzle XORs the
// slot with bits of the row so that those 8 rows x 2 slots land in distinct
// banks: bits 0-1 of the row (bit 1 for 8-slot rows, which pair up in one
// bank row) move the slot by 4, 8, 12, and bit 3 moves it by 2.
template <int S16>
__device__ __forceinline__ int w16_swz(int row) {
    static_assert(S16 == 16 || S16 == 8, "tile rows of 16 or 8 slots");
    if constexpr (S16 == 16) return ((row & 3) << 2) | (((row >> 3) & 1) << 1);
    else return (((row >> 1) & 1) << 2) | (((row >> 3) & 1) << 1);
}
template <int S16>
__device__ __forceinline__ int w16_off(int row, int slot) {
    return row * (S16 * 16) + ((slot ^ w16_swz<S16>(row)) << 4);
}

// MFMA operand (16 GEMM rows x 32 reduction values, bf16) from such a tile by
// two ds_read_b64_tr_b16: lane l gets GEMM row m0 + l % 16 (m0 a multiple of
// 16) and reduction values k0 + 8 (l / 16) .. +8.  In a group g of 16 lanes,
// lane j addresses reduction row k0 + 8 g + 4 h + j / 4 and GEMM columns
// m0 + 4 (j % 4) .. +4, so that lane i receives column m0 + i of four
// consecutive reduction rows (the read's lane mapping, see nat_frag_bf16).
template <int S16>
__device__ __forceinline__ v4u w16_frag_bf16(const char *tile, int k0, int m0, int lane) {
    const int g = lane >> 4, j = lane & 15;
    const int col = m0 + 4 * (j & 3);
    const int slot = col >> 3, within = (col & 7) * 2;
    v4u out;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int row = k0 + 8 * g + 4 * h + (j >> 2);
        const char *p = tile + w16_off<S16>(row, slot) + within;
        const v4s_t v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s_t *)(p));
        const v2u w = __builtin_bit_cast(v2u, v);
        out[2 * h] = w.x;
        out[2 * h + 1] = w.y;
    }
    return out;
}

// fp32 tiles (16-byte slots of 4 values; the swizzle XORs the slot with row
// bits 0-1, by 4, 8, 12): the operand of v_mfma_f32_16x16x4f32, lane l
// gets GEMM row m0 + l % 16 at reduction row k0 + l / 16 (one ds_read_b32;
// the 16 lanes of a group read 64 contiguous bytes of one row, the four
// groups four rows in distinct banks).
template <int S16>
__device__ __forceinline__ float f32_frag(const char *tile, int k0, int m0, int lane) {
    const int row = k0 + (lane >> 4), col = m0 + (lane & 15);
    return *reinterpret_cast<const float *>(tile + row * (S16 * 16) + (((col >> 2) ^ ((row & 3) << 2)) << 4) +
                                            (col & 3) * 4);
}

// The slot swizzle of a tile row: bf16 tiles the one of w16_off, fp32 tiles
// the one of f32_frag.
template <typename T, int S16>
__device__ __forceinline__ int tile_swz(int row) {
    if constexpr (sizeof(T) == 2) return w16_swz<S16>(row);
    else return (row & 3) << 2;
}

// T: uint16_t (bf16, 16x16x32 MFMAs, K steps of 32 pixels) or float (fp32,
// 16x16x4 fp32 MFMAs, K steps of 16 pixels); the tiles are the same bytes.
template <typename T, int BKP, int NS, int KG, int BO, bool SUM, bool LIN>
__device__ __forceinline__ void bwd_weight16_body(const BwdWeightArgs &a, char *smem_all) {
    // BO: output channels per term of the tile, 16 per wave (four or eight waves)
    constexpr bool BF = sizeof(T) == 2;
    constexpr int ES = (int)sizeof(T);
    constexpr int EPS = 16 / ES;        // elements per 16-byte slot
    constexpr int NT = BO * 4;          // threads of one pipeline
    constexpr int NTW = NT * KG;        // threads of the workgroup
    constexpr int KE = 64 / ES;         // output pixels per K step (one bf16 k-chunk, four fp32 ones)
    constexpr int SX = BKP / EPS;
    constexpr int SG = BO / EPS;
    constexpr int XB = KE * BKP * ES;
    constexpr int GB = KE * BO * ES;
    constexpr int STAGE = XB + 3 * GB;
    constexpr int NW = NT / 64;
    constexpr int NIX = XB / (NT * 16);
    constexpr int NIG = GB / (NT * 16);
    constexpr int NI = NIX + 3 * NIG;
    constexpr int RX = 64 / SX;
    constexpr int RG = 64 / SG;
    constexpr int MR = BKP / 16;        // 16-row k' fragments per wave
    constexpr int MH = MR / 2;          // ... per half step (register set)
    static_assert(XB % (NT * 16) == 0 && GB % (NT * 16) == 0 && MR % 2 == 0, "tile shape");
    static_assert(KG == 1 || KG == 2, "one or two pipelines");
    static_assert(BO == 64 || (BO == 128 && KG == 1), "four waves per pipeline, or eight in a single one");

    const int tid = threadIdx.x, lane = tid & 63;
    const int grp = KG == 1 ? 0 : wave_id() / NW, wave = KG == 1 ? wave_id() : wave_id() % NW;  // pipeline, wave in it
    char *const smem = smem_all + grp * (NS * STAGE);
    int bid = xcd_remap(blockIdx.x, gridDim.x);
    const int tiles = a.row_tiles * a.col_tiles;
    const int split = bid / tiles;
    bid -= split * tiles;
    const int rt = bid % a.row_tiles, ct = bid / a.row_tiles;
    // this pipeline's K steps: [s_begin, s_end); both pipelines run nst
    // iterations (the same barriers), the shorter one on zero-filled steps
    const int w_begin = split * a.stages_per_split;
    const int w_nst = min(a.stages_per_split, a.stages_total - w_begin);
    const int nst = (w_nst + KG - 1) / KG;
    const int s_begin = w_begin + grp * nst;
    const int s_end = min(s_begin + nst, w_begin + w_nst);

    const T *__restrict__ x = static_cast<const T *>(a.x);
    const T *__restrict__ gsrc[3] = {static_cast<const T *>(a.gy), static_cast<const T *>(a.ta),
                                     static_cast<const T *>(a.tb)};

    // DMA fill geometry (as in qconv_bwd_weight.h; the swizzle needs the tile
    // row mod 16 (bf16) or 4 (fp32), which instruction 0's row gives for every
    // instruction)
    constexpr int PHASE = BF ? 16 : 4;  // the rows the swizzle tells apart
    static_assert((RX * NW) % PHASE == 0 && (RG * NW) % PHASE == 0, "swizzle phase");
    const int xslot = (lane % SX) ^ tile_swz<T, SX>(RX * wave + lane / SX);
    const int kp = rt * BKP + EPS * xslot;
    const bool kp_ok = kp < a.KP;
    int xr, xq, xc;
    {
        const int tap = (int)fdiv((uint32_t)kp, a.fd_c);
        xc = kp - tap * a.C;
        xr = (int)fdiv((uint32_t)tap, a.fd_kw);
        xq = tap - xr * a.KW;
    }
    const int gslot = (lane % SG) ^ tile_swz<T, SG>(RG * wave + lane / SG);
    const int og = ct * BO + EPS * gslot;
    const bool og_ok = og < a.O;

    const int dh = xr - a.PH, dw = xq - a.PW;
    long long xlin[NIX], glin[NIG];
    int ohv[NIX], owv[NIX];
    if constexpr (LIN) {
#pragma unroll
        for (int i = 0; i < NIX; ++i) {
            const int m0 = s_begin * KE + RX * (NW * i + wave) + lane / SX;
            const int n = (int)fdiv((uint32_t)m0, a.fd_howo);
            const int rem = m0 - n * a.HO * a.WO;
            ohv[i] = (int)fdiv((uint32_t)rem, a.fd_wo);
            owv[i] = rem - ohv[i] * a.WO;
            xlin[i] = ((long long)m0 + (long long)dh * a.W + dw) * a.C + xc;
        }
#pragma unroll
        for (int i = 0; i < NIG; ++i)
            glin[i] = (long long)(s_begin * KE + RG * (NW * i + wave) + lane / SG) * a.O + og;
    }

    auto issue = [&](int s, int slot, bool live, int lo, int hi) {
        char *base = smem + slot * STAGE + wave * 1024;
        if constexpr (KG > 1) live = live && s < s_end;
        DmaPart part(lo, hi);
        if constexpr (LIN) {
            const int ds = s - s_begin;
            const int mleft = a.M - s * KE;
            const long long xs = (long long)ds * KE * a.C;
#pragma unroll
            for (int i = 0; i < NIX; ++i) {
                const int p = RX * (NW * i + wave) + lane / SX;
                const bool ok = live && kp_ok && p < mleft && (unsigned)(ohv[i] + dh) < (unsigned)a.H &&
                                (unsigned)(owv[i] + dw) < (unsigned)a.W;
                if (!part.take()) continue;
                dma16(dma_src(ok, x + (xlin[i] + xs), a.zero), base + i * (NT * 16));
                int ow = owv[i] + a.lin_dr;
                const int carry = ow >= a.WO ? 1 : 0;
                ow -= carry ? a.WO : 0;
                int oh = ohv[i] + a.lin_dq + carry;
                oh -= oh >= a.HO ? a.HO : 0;
                owv[i] = ow;
                ohv[i] = oh;
            }
            const long long gs = (long long)ds * KE * a.O;
#pragma unroll
            for (int i = 0; i < NIG; ++i) {
                const int p = RG * (NW * i + wave) + lane / SG;
                const bool ok = live && og_ok && p < mleft;
#pragma unroll
                for (int u = 0; u < 3; ++u)
                    if (part.take())
                        dma16(dma_src(ok, gsrc[u] + (glin[i] + gs), a.zero), base + XB + u * GB + i * (NT * 16));
            }
            return;
        }
#pragma unroll
        for (int i = 0; i < NIX; ++i) {
            const int m = s * KE + RX * (NW * i + wave) + lane / SX;
            const int n = (int)fdiv((uint32_t)m, a.fd_howo);
            const int rem = m - n * a.HO * a.WO;
            const int oh = (int)fdiv((uint32_t)rem, a.fd_wo);
            const int ow = rem - oh * a.WO;
            const int ih = oh * a.SH - a.PH + xr, iw = ow * a.SW - a.PW + xq;
            const bool ok = live && kp_ok && m < a.M && (unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W;
            if (part.take())
                dma16(dma_src(ok, x + ((size_t)(n * a.H + ih) * a.W + iw) * a.C + xc, a.zero), base + i * (NT * 16));
        }
#pragma unroll
        for (int i = 0; i < NIG; ++i) {
            const int m = s * KE + RG * (NW * i + wave) + lane / SG;
            const bool ok = live && og_ok && m < a.M;
            const size_t off = (size_t)m * a.O + og;
#pragma unroll
            for (int u = 0; u < 3; ++u)
                if (part.take()) dma16(dma_src(ok, gsrc[u] + off, a.zero), base + XB + u * GB + i * (NT * 16));
        }
    };

    f32x4_t acc[3][MR];
#pragma unroll
    for (int t = 0; t < 3; ++t)
#pragma unroll
        for (int mr = 0; mr < MR; ++mr) acc[t][mr] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
    float dsum[3] = {0.0f, 0.0f, 0.0f};

    const int ocol = wave * 16;  // this wave's 16 output channels within the tile
    // bf16 -- set 0: k' fragments 0 .. MH-1 and the G-side fragments; set 1: fragments MH .. MR-1.
    // fp32 -- set s: k-chunks 2 s, 2 s + 1 of the step, every k' fragment and the G-side values.
    v4u af[2][MH], gr[3], bt[3];
    float fa[2][2][MR], fg[2][2][3];
    auto read = [&](int slot, int ch, int set) {
        const char *xt = smem + slot * STAGE;
        if constexpr (BF) {
#pragma unroll
            for (int h = 0; h < MH; ++h) af[set][h] = w16_frag_bf16<SX>(xt, 0, (ch * MH + h) * 16, lane);
            if (ch == 0) {
#pragma unroll
                for (int u = 0; u < 3; ++u) gr[u] = w16_frag_bf16<SG>(xt + XB + u * GB, 0, ocol, lane);
            }
        } else {
#pragma unroll
            for (int kc = 0; kc < 2; ++kc) {
                const int k0 = 4 * (2 * ch + kc);
#pragma unroll
                for (int mr = 0; mr < MR; ++mr) fa[set][kc][mr] = f32_frag<SX>(xt, k0, mr * 16, lane);
#pragma unroll
                for (int u = 0; u < 3; ++u) fg[set][kc][u] = f32_frag<SG>(xt + XB + u * GB, k0, ocol, lane);
            }
        }
    };
    auto mma = [&](int set) {
        if constexpr (BF) {
            if (set == 0) {
                // the step's products, in fp32 (the bias sums use them before rounding), formed once
                float op[2][8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float gv = vget<T>(gr[0], e);
                    op[0][e] = gv * vget<T>(gr[2], e);
                    op[1][e] = gv * vget<T>(gr[1], e);
                }
                if constexpr (SUM) {
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        dsum[0] += op[0][e];
                        dsum[1] += op[1][e];
                        dsum[2] += vget<T>(gr[0], e);
                    }
                }
                bt[0] = vpack<T>(op[0]);
                bt[1] = vpack<T>(op[1]);
                bt[2] = gr[0];
            }
#pragma unroll
            for (int h = 0; h < MH; ++h)
#pragma unroll
                for (int t = 0; t < 3; ++t) mfma16(af[set][h], bt[t], acc[t][set * MH + h]);
        } else {
#pragma unroll
            for (int kc = 0; kc < 2; ++kc) {
                const float gv = fg[set][kc][0];
                const float op[3] = {gv * fg[set][kc][2], gv * fg[set][kc][1], gv};
                if constexpr (SUM) {
#pragma unroll
                    for (int t = 0; t < 3; ++t) dsum[t] += op[t];
                }
#pragma unroll
                for (int mr = 0; mr < MR; ++mr)
#pragma unroll
                    for (int t = 0; t < 3; ++t)
                        acc[t][mr] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[set][kc][mr], op[t], acc[t][mr], 0, 0, 0);
            }
        }
    };
    run_ring<NS, NI>(nst, s_begin, issue, read, mma);

    // Two pipelines: the second one's accumulators (and bias sums) go through
    // LDS into the first one's, lane for lane.
    if constexpr (KG == 2) {
        constexpr int NA = 3 * MR * 4;  // accumulator values per lane
        static_assert(4 * (NA + 3) * 64 * 4 <= KG * NS * STAGE, "exchange area fits");
        float *xch = reinterpret_cast<float *>(smem_all);
        lds_barrier();  // both rings are no longer read
        if (grp == 1) {
#pragma unroll
            for (int t = 0; t < 3; ++t)
#pragma unroll
                for (int mr = 0; mr < MR; ++mr)
#pragma unroll
                    for (int v = 0; v < 4; ++v) xch[(wave * NA + (t * MR + mr) * 4 + v) * 64 + lane] = acc[t][mr][v];
            if constexpr (SUM) {
#pragma unroll
                for (int t = 0; t < 3; ++t) xch[(4 * NA + wave * 3 + t) * 64 + lane] = dsum[t];
            }
        }
        lds_barrier();
        if (grp == 0) {
#pragma unroll
            for (int t = 0; t < 3; ++t)
#pragma unroll
                for (int mr = 0; mr < MR; ++mr)
#pragma unroll
                    for (int v = 0; v < 4; ++v) acc[t][mr][v] += xch[(wave * NA + (t * MR + mr) * 4 + v) * 64 + lane];
            if constexpr (SUM) {
#pragma unroll
                for (int t = 0; t < 3; ++t) dsum[t] += xch[(4 * NA + wave * 3 + t) * 64 + lane];
            }
        }
    }

    // dW epilogue (by the first pipeline's waves; every wave takes the
    // barriers and the stores): lane holds column o = ocol + lane % 16 of the
    // tile, rows k' = 16 mr + 4 (lane / 16) .. +4.  Staged through the idle
    // ring: each term's BO x BKP block (o rows, k' contiguous) goes out in
    // 16-byte chunks.
    const int lo = lane & 15, lg = lane >> 4;
    constexpr int PITCH = BKP * 4 + 16;
    constexpr int MAPB = BO * PITCH;
    constexpr int RING = KG * NS * STAGE;
    constexpr int PER = RING / MAPB >= 3 ? 3 : (RING / MAPB >= 1 ? RING / MAPB : 1);
    constexpr int CPR = BKP / 4;
    static_assert(MAPB <= RING, "staged dW tile fits the ring");
    const bool padded = a.C_out != a.C;
    const int KPO = a.KH * a.KW * a.C_out;
    const bool vec_out = (a.KP & 3) == 0 && !padded;
    if (vec_out) {
#pragma unroll
        for (int t0 = 0; t0 < 3; t0 += PER) {
            lds_barrier();
#pragma unroll
            for (int t = t0; t < t0 + PER && t < 3; ++t) {
                char *tile = smem_all + (t - t0) * MAPB;
                if (grp != 0) continue;
#pragma unroll
                for (int mr = 0; mr < MR; ++mr) {
                    const int kl = mr * 16 + 4 * lg;
                    store4<float>(reinterpret_cast<float *>(tile + (ocol + lo) * PITCH + kl * 4), acc[t][mr][0],
                                  acc[t][mr][1], acc[t][mr][2], acc[t][mr][3]);
                }
            }
            lds_barrier();
#pragma unroll
            for (int t = t0; t < t0 + PER && t < 3; ++t) {
                const char *tile = smem_all + (t - t0) * MAPB;
                float *__restrict__ dst =
                    a.splits == 1 ? a.dw[t] : a.ws_dw + ((size_t)split * 3 + t) * (size_t)a.O * KPO;
                for (int c = tid; c < BO * CPR; c += NTW) {
                    const int row = c / CPR, cc = c % CPR;
                    const int o = ct * BO + row, k = rt * BKP + 4 * cc;
                    if (o < a.O && k < a.KP)
                        *reinterpret_cast<v4u *>(dst + (size_t)o * a.KP + k) = lds_read16(tile + row * PITCH + cc * 16);
                }
            }
        }
    } else if (grp == 0) {
#pragma unroll
        for (int t = 0; t < 3; ++t) {
            float *__restrict__ dst = a.splits == 1 ? a.dw[t] : a.ws_dw + ((size_t)split * 3 + t) * (size_t)a.O * KPO;
            const int o = ct * BO + ocol + lo;
            if (o >= a.O) continue;
#pragma unroll
            for (int mr = 0; mr < MR; ++mr) {
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int kk = rt * BKP + mr * 16 + 4 * lg + v;
                    if (kk >= a.KP) continue;
                    if (!padded) {
                        dst[(size_t)o * a.KP + kk] = acc[t][mr][v];
                    } else {
                        const int tap = (int)fdiv((uint32_t)kk, a.fd_c);
                        const int c = kk - tap * a.C;
                        if (c < a.C_out) dst[(size_t)o * KPO + tap * a.C_out + c] = acc[t][mr][v];
                    }
                }
            }
        }
    }

    // Bias gradients: the four lane groups hold the pixel quarters of channel lane % 16.
    if (SUM && grp == 0) {
#pragma unroll
        for (int t = 0; t < 3; ++t) {
            float tot = dsum[t] + __shfl_xor(dsum[t], 16);
            tot += __shfl_xor(tot, 32);
            const int o = ct * BO + ocol + lo;
            if (lg == 0 && o < a.O) {
                if (a.splits == 1)
                    a.db[t][o] = tot;
                else
                    a.ws_db[((size_t)split * 3 + t) * a.O + o] = tot;
            }
        }
    }
}

template <int BKP, int NS, int KG = 1, int BO = 64, typename T = uint16_t>
__global__ __launch_bounds__(BO * 4 * KG) void qconv_bwd_weight16_kernel(const BwdWeightArgs a) {
    constexpr int STAGE = 64 * BKP + 3 * 64 * BO;  // a K step: 64 bytes of every X and G-side tile row
    __shared__ __attribute__((aligned(1024))) char smem[KG * NS * STAGE];
    int bid = xcd_remap(blockIdx.x, gridDim.x);
    const int tiles = a.row_tiles * a.col_tiles;
    bid -= (bid / tiles) * tiles;
    const bool sum = a.want_db && bid % a.row_tiles == 0;
    if (a.lin) {
        if (sum) bwd_weight16_body<T, BKP, NS, KG, BO, true, true>(a, smem);
        else bwd_weight16_body<T, BKP, NS, KG, BO, false, true>(a, smem);
    } else {
        if (sum) bwd_weight16_body<T, BKP, NS, KG, BO, true, false>(a, smem);
        else bwd_weight16_body<T, BKP, NS, KG, BO, false, false>(a, smem);
    }
}

}  // namespace ql
