// qconv_fwd_ksplit.h -- forward of the quadratic convolution layer (arXiv
// 2204.01701, section 3.1, eq:2ndneuron3) for layers whose output is too
// small to fill the GPU with the tiled kernel's workgroup tiles: the 4 x 4 and
// 2 x 2 maps of a CIFAR VGG-16 (512 to 2048 output pixels, 512 channels,
// K = 2304 to 4608).
//
// The tiled kernel (qconv_fwd.h) covers such a layer with 32 to 128 tiles and
// splits K over workgroups, whose raw fp32 partials of all three terms then
// go through HBM to a combine kernel.  Here a workgroup's tile is small
// (3 x 16 RB weight rows by 16 CB pixels), so that the tiles alone fill the
// GPU, and the four waves of the workgroup split the tile's K range:
//   - each wave copies its chunks (32 bf16 or 16 fp32 reduction values
//     within one tap: 64 contiguous bytes of each OHWI weight row and of each
//     pixel's NHWC channels) into a private LDS ring with buffer loads, one
//     coalesced instruction per 16-row fragment (the swizzled 64-byte-row
//     layout of qpipe.h), and reads each MFMA operand back as one 16-byte
//     run per lane; its waits are its own (vmcnt, lgkmcnt), with no barrier
//     in the loop;
//   - the waves' fp32 accumulators are then added through LDS in wave order
//     (a fixed order, so results are bitwise repeatable), and each wave
//     finishes its share of the tile's 16 x 16 blocks: the biases,
//     Y = T_a o T_b + T_c, the fused scale / shift / ReLU and statistics, the
//     stores of Y, T_a and T_b.  No term map leaves the chip unfinished.
// The K range of a tile is its in-bounds taps only (the union over its
// pixels).  With the position-major pixel order (FwdArgs::pm) the pixels of
// a tile share one output position, so on a padded 2 x 2 map 5 of the 9 taps
// of a 3 x 3 filter drop out of every tile.
#pragma once

#include "qargs.h"
#include "qdevice.h"
#include "qconv_fwd_narrow.h"
#include "qpipe.h"

namespace ql {

// Taps of the filter in bounds for GEMM column m (bit r KW + q).
__device__ __forceinline__ uint32_t fwd_column_taps(const FwdArgs &a, int m) {
    int pos;
    if (a.pm) {
        pos = (int)fdiv((uint32_t)m, a.fd_n);
    } else {
        const int n = (int)fdiv((uint32_t)m, a.fd_howo);
        pos = m - n * a.HO * a.WO;
    }
    const int oh = (int)fdiv((uint32_t)pos, a.fd_wo);
    const int h0 = oh * a.SH - a.PH, w0 = (pos - oh * a.WO) * a.SW - a.PW;
    uint32_t u = 0;
    for (int r = 0; r < a.KH; ++r)
        for (int q = 0; q < a.KW; ++q)
            if ((unsigned)(h0 + r) < (unsigned)a.H && (unsigned)(w0 + q) < (unsigned)a.W) u |= 1u << (r * a.KW + q);
    return u;
}

// RB: 16-channel row blocks per term, CB: 16-pixel column blocks (RB CB a
// multiple of the four waves, at most 64 pixels), NS: ring stages per wave.
// C is a multiple of the chunk (narrow_chunk), so a chunk lies within one
// tap; O a multiple of 4.
template <typename T, int RB, int CB, int NS, bool EPI>
__global__ __launch_bounds__(kThreads, 4 * NS * (3 * RB + CB) * 1024 > 80 * 1024 ? 1 : 2) void qconv_fwd_ksplit_kernel(
    const FwdArgs a) {
    constexpr int CK = narrow_chunk<T>();
    constexpr int VEC = Elem<T>::VEC;
    constexpr int NWV = kThreads / 64;
    constexpr int NB = RB * CB;
    constexpr int BCOL = 16 * CB;
    constexpr int NF = 3 * RB + CB;       // 16-row fragments (1 KB of LDS each) per chunk
    constexpr int STAGE = NF * 1024;
    constexpr int XCH = NWV * NWV * 3 * 4 * 64 * 4;  // the reduction's exchange area (bytes)
    constexpr int LDS = NWV * NS * STAGE > XCH ? NWV * NS * STAGE : XCH;
    static_assert(NWV == 4 && NB % NWV == 0 && BCOL <= 64 && NS >= 2, "tile shape");
    static_assert((NS - 2) * NF < 64, "vmcnt range");
    __shared__ __attribute__((aligned(1024))) char smem[LDS];

    const int lane = threadIdx.x & 63, li = lane & 15, lg = lane >> 4;
    const int wave = wave_id();
    const int bid = xcd_remap(blockIdx.x, gridDim.x);
    const int rt = bid / a.col_tiles, ct = bid - rt * a.col_tiles;
    const int o0 = rt * 16 * RB, m0 = ct * BCOL;
    constexpr int ES = (int)sizeof(T);
    // Buffer resources of X and the weights (byte offsets of 32 bits: the
    // planner keeps both below 2^31 bytes); an offset past the end reads zeros.
    const __amdgpu_buffer_rsrc_t xrs = raw_rsrc(a.x, (uint32_t)a.N * a.H * a.W * a.C * ES);
    const uint32_t wbytes = (uint32_t)a.O * a.K * ES;
    const __amdgpu_buffer_rsrc_t wrs[3] = {raw_rsrc(a.w[0], wbytes), raw_rsrc(a.w[1], wbytes),
                                           raw_rsrc(a.w[2], wbytes)};
    char *const ring = smem + wave * (NS * STAGE);

    // The tile's taps: lane l < BCOL takes column m0 + l, the wave ORs them.
    uint32_t tmask = 0;
    if (lane < BCOL && m0 + lane < a.M) tmask = fwd_column_taps(a, m0 + lane);
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) tmask |= (uint32_t)__shfl_xor((int)tmask, d);
    tmask = __builtin_amdgcn_readfirstlane(tmask);
    // This wave's chunks [k0, k1) of the tile's popcount(tmask) cps chunks.
    const int nchunks = __builtin_popcount(tmask) * a.cps;
    const int k0 = wave * nchunks / NWV, k1 = (wave + 1) * nchunks / NWV;

    // DMA geometry: one instruction fills a fragment's 64 LDS slots, lane l
    // the slot of row l / 4 and logical 16-byte column dcol (the KM layout of
    // qpipe.h, whose swizzle puts the fragment reads of 16 consecutive rows in
    // distinct bank groups).  A: weight row o = o0 + 16 rb + l / 4, its byte
    // offset fixed per lane (rows past O re-read row O - 1: their results are
    // never stored), the chunk's offset a scalar.
    const int drow = lane >> 2, dcol = km_fill_col(lane);
    uint32_t woff[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        const int o = o0 + 16 * rb + drow;
        woff[rb] = (uint32_t)((min(o, a.O - 1) * a.K + VEC * dcol) * ES);
    }
    // B: column m = m0 + 16 cb + l / 4: the window origin (ih0, iw0) of its
    // pixel and the element offset of that origin's run dcol; columns past M
    // and taps in the padding read zeros (an out-of-range offset).
    int xoff[CB], xh[CB], xw[CB];
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) {
        const int m = m0 + 16 * cb + drow;
        const bool mok = m < a.M;
        const int mm = mok ? m : a.M - 1;
        int n, pos;
        if (a.pm) {
            pos = (int)fdiv((uint32_t)mm, a.fd_n);
            n = mm - pos * a.N;
        } else {
            n = (int)fdiv((uint32_t)mm, a.fd_howo);
            pos = mm - n * a.HO * a.WO;
        }
        const int oh = (int)fdiv((uint32_t)pos, a.fd_wo);
        xh[cb] = mok ? oh * a.SH - a.PH : -(1 << 20);  // (no tap brings it in bounds)
        xw[cb] = (pos - oh * a.WO) * a.SW - a.PW;
        xoff[cb] = ((n * a.H + oh * a.SH - a.PH) * a.W + xw[cb]) * a.C + VEC * dcol;
    }

    // Chunk state (wave-uniform): channel chunk cc of tap `tap` = (tr, tq); `rest`
    // holds the taps not yet finished, the current one its lowest bit.
    const int ti0 = (int)fdiv((uint32_t)k0, a.fd_cps);
    int cc = k0 - ti0 * a.cps;
    uint32_t rest = tmask;
    for (int i = 0; i < ti0; ++i) rest &= rest - 1;
    int tap = rest ? __builtin_ctz(rest) : 0;
    int tr = (int)fdiv((uint32_t)tap, a.fd_kw), tq = tap - tr * a.KW;

    // Copy the current chunk into ring slot `slot`, then step to the next chunk.
    // (Chunks past the wave's range, copied to keep the ring's count of copies
    // fixed, are never read into an MFMA.)
    auto issue = [&](int slot) {
        char *base = ring + slot * STAGE;
        const int kw = (tap * a.C + cc * CK) * ES;
#pragma unroll
        for (int t = 0; t < 3; ++t)
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) dma16_buf(wrs[t], woff[rb], kw, base + (t * RB + rb) * 1024);
        const int kx = (tr * a.W + tq) * a.C + cc * CK;
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) {
            const bool ok = (unsigned)(xh[cb] + tr) < (unsigned)a.H && (unsigned)(xw[cb] + tq) < (unsigned)a.W;
            dma16_buf(xrs, ok ? (uint32_t)((xoff[cb] + kx) * ES) : 0x80000000u, 0, base + (3 * RB + cb) * 1024);
        }
        if (++cc == a.cps) {
            cc = 0;
            rest &= rest - 1;
            tap = rest ? __builtin_ctz(rest) : 0;
            tr = (int)fdiv((uint32_t)tap, a.fd_kw);
            tq = tap - tr * a.KW;
        }
    };
    // The MFMA operand of lane (li, lg): row li, logical column lg of a fragment.
    const int foff = km_off(li, lg);
    auto read = [&](int slot, v4u (&fa)[3][RB], v4u (&fb)[CB]) {
        const char *base = ring + slot * STAGE;
#pragma unroll
        for (int t = 0; t < 3; ++t)
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) fa[t][rb] = lds_read16(base + (t * RB + rb) * 1024 + foff);
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) fb[cb] = lds_read16(base + (3 * RB + cb) * 1024 + foff);
    };
    f32x4n_t acc[3][RB][CB];
#pragma unroll
    for (int t = 0; t < 3; ++t)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
            for (int cb = 0; cb < CB; ++cb) acc[t][rb][cb] = f32x4n_t{0.0f, 0.0f, 0.0f, 0.0f};
    auto mma = [&](const v4u (&fa)[3][RB], const v4u (&fb)[CB]) {
#pragma unroll
        for (int t = 0; t < 3; ++t)
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                for (int cb = 0; cb < CB; ++cb) narrow_mfma<T>(fa[t][rb], fb[cb], acc[t][rb][cb]);
    };

    // The wave's ring: chunk j in slot j % NS, NS chunks in flight.  Step k (the
    // fragments of chunk k already in registers): the MFMAs of chunk k; wait
    // for chunk k + 1's copies and for the fragment reads (so chunk k's slot
    // is free); copy chunk k + NS into chunk k's slot; read chunk k + 1's
    // fragments.  Only this wave touches its ring, so the waits are per wave
    // (vmcnt, lgkmcnt) and there is no barrier; the copies are asm the
    // compiler cannot order against LDS reads, hence the explicit waits with
    // memory clobbers.  (One register set: the reads of chunk k + 1 overlap the
    // MFMAs of chunk k in the matrix pipeline.)
    constexpr int VMC = (NS - 1) * NF;
    constexpr int VM_IMM = (VMC & 15) | ((VMC >> 4) << 14) | (7 << 4) | (15 << 8);
#pragma unroll
    for (int j = 0; j < NS; ++j) issue(j);
    v4u fa[3][RB], fb[CB];
    constexpr int VM0 = (NS - 1) * NF;
    __builtin_amdgcn_s_waitcnt((VM0 & 15) | ((VM0 >> 4) << 14) | (7 << 4) | (15 << 8));  // chunk k0 landed
    asm volatile("" ::: "memory");
    read(0, fa, fb);
    int slot = 0;  // chunk k's slot
    for (int k = k0; k < k1; ++k) {
        mma(fa, fb);
        const int s1 = slot + 1 == NS ? 0 : slot + 1;
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // chunk k's fragments read
        issue(slot);
        __builtin_amdgcn_s_waitcnt(VM_IMM);  // chunk k + 1 landed
        asm volatile("" ::: "memory");
        read(s1, fa, fb);
        slot = s1;
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // no copy into the ring still in flight
    __syncthreads();  // every wave done with its ring: the exchange area overlaps them
    float *const xch = reinterpret_cast<float *>(smem);

    // The waves' sums, block by block in phases of four blocks: wave w
    // finishes block 4 ph + w of phase ph, adding the four partials in wave order.
    T *__restrict__ y = static_cast<T *>(a.y);
    T *__restrict__ ta = static_cast<T *>(a.ta);
    T *__restrict__ tb = static_cast<T *>(a.tb);
    const bool stats = EPI && a.stat_part != nullptr;
#pragma unroll
    for (int ph = 0; ph < NB / NWV; ++ph) {
        if (ph > 0) __syncthreads();  // the previous phase's reads are done
#pragma unroll
        for (int j = 0; j < NWV; ++j) {
            const int blk = ph * NWV + j, rb = blk / CB, cb = blk % CB;
#pragma unroll
            for (int t = 0; t < 3; ++t)
#pragma unroll
                for (int v = 0; v < 4; ++v) xch[(((wave * NWV + j) * 3 + t) * 4 + v) * 64 + lane] = acc[t][rb][cb][v];
        }
        __syncthreads();
        const int blk = ph * NWV + wave, rb = blk / CB, cb = blk % CB;
        float s[3][4];
#pragma unroll
        for (int t = 0; t < 3; ++t)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                float sum = 0.0f;
#pragma unroll
                for (int src = 0; src < NWV; ++src) sum += xch[(((src * NWV + wave) * 3 + t) * 4 + v) * 64 + lane];
                s[t][v] = sum;
            }
        // Epilogue of the block: lane holds column m, channels o .. o + 3.
        const int m = m0 + 16 * cb + li;
        const int o = o0 + 16 * rb + 4 * lg;
        const bool live = m < a.M && o < a.O;
        float ssum[4] = {0.0f, 0.0f, 0.0f, 0.0f}, ssq[4] = {0.0f, 0.0f, 0.0f, 0.0f};
        if (live) {
            float va[4], vb[4], yv[4];
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                va[v] = s[0][v] + (a.bias[0] ? a.bias[0][o + v] : 0.0f);
                vb[v] = s[1][v] + (a.bias[1] ? a.bias[1][o + v] : 0.0f);
                const float vc = s[2][v] + (a.bias[2] ? a.bias[2][o + v] : 0.0f);
                yv[v] = va[v] * vb[v] + vc;
                if constexpr (EPI) yv[v] = epi_apply(a.epi, o + v, yv[v]);
            }
            int row = m;  // NHWC row of column m
            if (a.pm) {
                const int pos = (int)fdiv((uint32_t)m, a.fd_n);
                row = (m - pos * a.N) * a.HO * a.WO + pos;
            }
            const size_t off = (size_t)row * a.O + o;
            if (y) store4<T>(y + off, yv[0], yv[1], yv[2], yv[3]);
            if (ta) store4<T>(ta + off, va[0], va[1], va[2], va[3]);
            if (tb) store4<T>(tb + off, vb[0], vb[1], vb[2], vb[3]);
            if (stats) {
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const float f = to_f32<T>(from_f32<T>(yv[v]));  // the stored value
                    ssum[v] = f;
                    ssq[v] = f * f;
                }
            }
        }
        if (stats) {
            // part ct CB + cb of the statistics: the block's 16 columns, added in a fixed butterfly
            float *part = a.stat_part + (size_t)(ct * CB + cb) * 2 * a.O;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                float s1 = ssum[v], s2 = ssq[v];
#pragma unroll
                for (int d = 1; d < 16; d <<= 1) {
                    s1 += __shfl_xor(s1, d);
                    s2 += __shfl_xor(s2, d);
                }
                if (li == 0 && o < a.O) {
                    part[o + v] = s1;
                    part[a.O + o + v] = s2;
                }
            }
        }
    }
}

}  // namespace ql
