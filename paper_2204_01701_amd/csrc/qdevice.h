// qdevice.h -- device helpers shared by the quadratic-layer kernels (gfx950 only).
//
// Element types: float (fp32) or uint16_t holding bfloat16 bits.  Every LDS
// operand tile is stored "K-contiguous": one row per GEMM row/column, the
// reduction index contiguous inside the row, padded by 16 bytes so that the
// 16-byte fragment reads of the MFMA operands are bank-conflict free.  A
// "chunk" is 32 bytes of one row: 16 bf16 (one v_mfma_f32_32x32x16_bf16) or
// 8 fp32 (four v_mfma_f32_32x32x2_f32).  Lane l of a wave reads the 16 bytes
// at offset (l / 32) * 16 of row (l % 32) of a 32-row block.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "qfastdiv.h"
#include "qargs.h"

namespace ql {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t v4u __attribute__((ext_vector_type(4)));  // 16 raw bytes
typedef uint32_t v2u __attribute__((ext_vector_type(2)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;  // 4 waves of 64 lanes per workgroup

__device__ __forceinline__ uint32_t fdiv(uint32_t n, const FastDiv &f) {
    return (uint32_t)(((uint64_t)__umulhi(n, f.m) + n) >> f.s);
}

// ---------------------------------------------------------------------------
// Element traits and conversions.
// ---------------------------------------------------------------------------
template <typename T> struct Elem;
template <> struct Elem<float> {
    static constexpr int VEC = 4;  // elements per 16 bytes
};
template <> struct Elem<uint16_t> {
    static constexpr int VEC = 8;
};

__device__ __forceinline__ float bf2f(uint32_t bits16) { return __uint_as_float(bits16 << 16); }

// Round-to-nearest-even conversion of two floats into one dword of bf16 (lo = a).
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
    bf16x2_t v = {(__bf16)a, (__bf16)b};
    return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ uint16_t f2bf(float a) { return __builtin_bit_cast(uint16_t, (__bf16)a); }

// Element e (0..VEC-1) of a 16-byte vector as float.
template <typename T> __device__ __forceinline__ float vget(const v4u &v, int e);
template <> __device__ __forceinline__ float vget<float>(const v4u &v, int e) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    return __uint_as_float(w[e]);
}
template <> __device__ __forceinline__ float vget<uint16_t>(const v4u &v, int e) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    return bf2f((w[e >> 1] >> ((e & 1) * 16)) & 0xffffu);
}

// Pack VEC floats into a 16-byte vector of T.
template <typename T> __device__ __forceinline__ v4u vpack(const float *f);
template <> __device__ __forceinline__ v4u vpack<float>(const float *f) {
    return v4u{__float_as_uint(f[0]), __float_as_uint(f[1]), __float_as_uint(f[2]), __float_as_uint(f[3])};
}
template <> __device__ __forceinline__ v4u vpack<uint16_t>(const float *f) {
    return v4u{pack_bf16x2(f[0], f[1]), pack_bf16x2(f[2], f[3]), pack_bf16x2(f[4], f[5]),
                      pack_bf16x2(f[6], f[7])};
}

// Raw 16-bit / 32-bit element access without conversion (for transposes).
template <typename T> __device__ __forceinline__ uint32_t vraw(const v4u &v, int e) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    if constexpr (sizeof(T) == 4) {
        return w[e];
    } else {
        return (w[e >> 1] >> ((e & 1) * 16)) & 0xffffu;
    }
}

// Wave-local ordering of LDS writes before reads of other lanes of the wave.
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// The forward epilogue of output channel o (EpiArgs): scale, shift, ReLU.
__device__ __forceinline__ float epi_apply(const EpiArgs &e, int o, float v) {
    if (e.scale) v *= e.scale[o];
    if (e.shift) v += e.shift[o];
    return e.relu ? fmaxf(v, 0.0f) : v;
}

template <typename T> __device__ __forceinline__ float to_f32(T v);
template <> __device__ __forceinline__ float to_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f32<uint16_t>(uint16_t v) { return bf2f(v); }

template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ uint16_t from_f32<uint16_t>(float v) { return f2bf(v); }

// Store 4 consecutive values (fp32 in registers) as T: 16 B for fp32, 8 B for bf16.
template <typename T> __device__ __forceinline__ void store4(T *p, float a, float b, float c, float d);
template <> __device__ __forceinline__ void store4<float>(float *p, float a, float b, float c, float d) {
    *reinterpret_cast<v4f *>(p) = v4f{a, b, c, d};
}
template <> __device__ __forceinline__ void store4<uint16_t>(uint16_t *p, float a, float b, float c, float d) {
    *reinterpret_cast<v2u *>(p) = v2u{pack_bf16x2(a, b), pack_bf16x2(c, d)};
}

// ---------------------------------------------------------------------------
// MFMA on one 32-byte chunk: acc(32x32) += A(32 x chunk) * B(chunk x 32).
// a, b: the 16 bytes this lane holds of the A row (lane % 32) and B column
// (lane % 32).  Output layout: lane l holds column l % 32 and rows
// 8 * (v / 4) + 4 * (l / 32) + (v % 4), v = 0..15.
// ---------------------------------------------------------------------------
template <typename T> __device__ __forceinline__ void mfma_chunk(const v4u &a, const v4u &b, f32x16_t &acc);

template <> __device__ __forceinline__ void mfma_chunk<uint16_t>(const v4u &a, const v4u &b, f32x16_t &acc) {
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                  acc, 0, 0, 0);
}

template <> __device__ __forceinline__ void mfma_chunk<float>(const v4u &a, const v4u &b, f32x16_t &acc) {
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
}

// Products of the prologue on one 16-byte fragment: G o T_b and G o T_a.
template <typename T>
__device__ __forceinline__ void prologue_frag(const v4u &g, const v4u &ta, const v4u &tb, v4u &ga, v4u &gb) {
    constexpr int VEC = Elem<T>::VEC;
    float fa[VEC], fb[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
        const float gv = vget<T>(g, e);
        fa[e] = gv * vget<T>(tb, e);
        fb[e] = gv * vget<T>(ta, e);
    }
    ga = vpack<T>(fa);
    gb = vpack<T>(fb);
}

// Elementwise square of a 16-byte fragment (fp32 products rounded once to T):
// the X o X operand of the T2 neuron.
template <typename T> __device__ __forceinline__ v4u square_frag(const v4u &v) {
    constexpr int VEC = Elem<T>::VEC;
    float f[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
        const float x = vget<T>(v, e);
        f[e] = x * x;
    }
    return vpack<T>(f);
}

// The output-side MFMA operands of a backward kernel for operand mode OM
// (qargs.h), formed in fp32 on one 16-byte fragment of G, T_a, T_b and
// rounded once to T:
//   OM_QUADRA, OM_QSQ: G o T_b, G o T_a, G      OM_PAIR: G o T_b, G o T_a
//   OM_SQUARE: 2 G o T_a                        OM_SQIN: G
template <typename T, int OM>
__device__ __forceinline__ void operands_frag(const v4u &g, const v4u &ta, const v4u &tb, v4u *bt) {
    constexpr int VEC = Elem<T>::VEC;
    if constexpr (OM == OM_SQIN) {
        bt[0] = g;
    } else if constexpr (OM == OM_SQUARE) {
        float f[VEC];
#pragma unroll
        for (int e = 0; e < VEC; ++e) f[e] = 2.0f * vget<T>(g, e) * vget<T>(ta, e);
        bt[0] = vpack<T>(f);
    } else {
        prologue_frag<T>(g, ta, tb, bt[0], bt[1]);
        if constexpr (om_three(OM)) bt[2] = g;
    }
}

// Four consecutive elements of T as floats (8 bytes for bf16, 16 for fp32).
template <typename T> __device__ __forceinline__ void load4(const T *p, float *f) {
    if constexpr (sizeof(T) == 4) {
        const v4f v = *reinterpret_cast<const v4f *>(p);
        f[0] = v[0]; f[1] = v[1]; f[2] = v[2]; f[3] = v[3];
    } else {
        const v2u v = *reinterpret_cast<const v2u *>(p);
        f[0] = bf2f(v.x & 0xffffu); f[1] = bf2f(v.x >> 16);
        f[2] = bf2f(v.y & 0xffffu); f[3] = bf2f(v.y >> 16);
    }
}

// Input-gradient epilogue of the T4 + identity and T2 neurons on a wave's
// accumulator tile (rows: input channels c, columns: input pixels m, the MFMA
// layout of mfma_chunk): acc += src[m, c] (src = G, the shortcut's gradient)
// or acc *= 2 src[m, c] (src = X, the derivative of X o X).  src is M x C.
template <typename T, int OM, int MR, int MC>
__device__ __forceinline__ void neuron_dx_epilogue(f32x16_t (&acc)[MR][MC], const void *srcv, int M, int C,
                                                   int pcol0, int crow0, int lane) {
    const T *__restrict__ src = static_cast<const T *>(srcv);
    const int lrow = lane & 31, lhi = lane >> 5;
#pragma unroll
    for (int mr = 0; mr < MR; ++mr)
#pragma unroll
        for (int mc = 0; mc < MC; ++mc) {
            const int m = pcol0 + mc * 32 + lrow;
            if (m >= M) continue;
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int c = crow0 + mr * 32 + 8 * g + 4 * lhi;
                float v[4] = {0.0f, 0.0f, 0.0f, 0.0f};
                if ((C & 3) == 0 && c < C) {
                    load4<T>(src + (size_t)m * C + c, v);  // four channels in one load
                } else {
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        if (c + i < C) v[i] = to_f32<T>(src[(size_t)m * C + c + i]);
                }
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float r = acc[mr][mc][4 * g + i];
                    acc[mr][mc][4 * g + i] = OM == OM_SQIN ? r * (2.0f * v[i]) : r + v[i];
                }
            }
        }
}

// Input-gradient epilogue of the T2&4 neuron: the terms a, b accumulated in
// acc, the c term (whose operand is X o X) in acc2; acc += 2 X[m, c] acc2
// (the chain rule through the square).  X is M x C.  Linear in the
// accumulators, so each split-K partial may take it before the sum.
template <typename T, int MR, int MC>
__device__ __forceinline__ void qsq_dx_epilogue(f32x16_t (&acc)[MR][MC], const f32x16_t (&acc2)[MR][MC],
                                                const void *xv, int M, int C, int pcol0, int crow0, int lane) {
    const T *__restrict__ x = static_cast<const T *>(xv);
    const int lrow = lane & 31, lhi = lane >> 5;
#pragma unroll
    for (int mr = 0; mr < MR; ++mr)
#pragma unroll
        for (int mc = 0; mc < MC; ++mc) {
            const int m = pcol0 + mc * 32 + lrow;
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int c = crow0 + mr * 32 + 8 * g + 4 * lhi;
                float v[4] = {0.0f, 0.0f, 0.0f, 0.0f};
                if (m < M) {
                    if ((C & 3) == 0 && c < C) {
                        load4<T>(x + (size_t)m * C + c, v);
                    } else {
#pragma unroll
                        for (int i = 0; i < 4; ++i)
                            if (c + i < C) v[i] = to_f32<T>(x[(size_t)m * C + c + i]);
                    }
                }
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    acc[mr][mc][4 * g + i] += (2.0f * v[i]) * acc2[mr][mc][4 * g + i];
            }
        }
}

// 16-byte global load, or zeros when !ok (the address is not touched then).
template <typename P> __device__ __forceinline__ v4u ld16(const P *p, bool ok) {
    v4u v = {0u, 0u, 0u, 0u};
    if (ok) v = *reinterpret_cast<const v4u *>(p);
    return v;
}

__device__ __forceinline__ v4u lds_read16(const char *p) { return *reinterpret_cast<const v4u *>(p); }
__device__ __forceinline__ void lds_write16(char *p, const v4u &v) { *reinterpret_cast<v4u *>(p) = v; }

// Workgroups are dispatched round-robin over the 8 XCDs (each with its own
// L2).  Remap the hardware order so that each XCD receives a contiguous range
// of logical tiles: tiles that share an operand then share an L2.
__device__ __forceinline__ int xcd_remap(int bid, int nblk) {
    const int full = nblk & ~7;
    if (bid >= full) return bid;
    return (bid & 7) * (full >> 3) + (bid >> 3);
}

// Logical block -> (split, row tile, column tile) of a split-K grid, in one of
// three orders; with xcd_remap, the order decides what the blocks of one XCD
// share, and so which operand each XCD reads whole from beyond its L2:
//   0 split-major   (split, column tile, row tile): a K range;
//   1 tile-major    (column tile, row tile, split): output tiles, all K;
//   2 row-major     (row tile, split, column tile): the K rows of a row tile.
struct TileCoord {
    int split, rt, ct;
};
__device__ __forceinline__ TileCoord tile_coord(int bid, int order, int row_tiles, int col_tiles, int splits) {
    TileCoord c;
    if (order == 1) {
        c.split = bid % splits;
        bid /= splits;
        c.rt = bid % row_tiles;
        c.ct = bid / row_tiles;
    } else if (order == 2) {
        const int per = splits * col_tiles;
        c.rt = bid / per;
        bid -= c.rt * per;
        c.split = bid / col_tiles;
        c.ct = bid - c.split * col_tiles;
    } else {
        const int tiles = row_tiles * col_tiles;
        c.split = bid / tiles;
        bid -= c.split * tiles;
        c.rt = bid % row_tiles;
        c.ct = bid / row_tiles;
    }
    return c;
}

}  // namespace ql
