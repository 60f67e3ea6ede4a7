// qlaunch_bwd_data.hip -- launches of the input-gradient kernels (pipelined, wide, few-channel column kernels, generic, split reduction).
#include "qhost.h"
#include "qconv_bwd_data.h"
#include "qconv_bwd_data_wide.h"
#include "qconv_bwd_data_narrow.h"
#include "qconv_generic.h"

namespace ql {
namespace host {

// xin: X, for the types whose terms see X o X (T2, T2&4), else unused.
template <typename T>
ql_status launch_bwd_data(const Geom &g, const BwdDataPlan &p, const void *gy, const void *ta, const void *tb,
                          const void *xin, const void *wa, const void *wb, const void *wc, void *dx, void *ws,
                          hipStream_t st) {
    if (p.smallc && p.fused_rb) {
        const int bands = cdiv(g.H, p.fused_rb);
#define QL_BD_FUSED(NT)                                                                                            \
    hipLaunchKernelGGL((qconv_bwd_data_cols_fused_kernel<T, NT>), dim3(g.N * bands), dim3(NT), p.fused_smem, st,    \
                       static_cast<const T *>(gy), static_cast<const T *>(ta), static_cast<const T *>(tb),          \
                       static_cast<const T *>(wa), static_cast<const T *>(wb), static_cast<const T *>(wc),          \
                       static_cast<T *>(dx), g.H, g.W, g.C, g.O, g.KH, g.KW, g.PH, g.PW, g.HO, g.WO, p.fused_rb, \
                       (int)(p.smem / sizeof(v4u)))
        // 8 waves: each takes one or two 32-pixel groups of the band (measured faster than 4)
        if (env_override("QLAYER_BWD_DATA_FUSED_NT", 512) == 256)
            QL_BD_FUSED(256);
        else
            QL_BD_FUSED(512);
#undef QL_BD_FUSED
        return hip_status();
    }
    if (p.smallc) {
        const long long Mo = (long long)g.N * g.HO * g.WO;
        const int J = g.KH * g.KW * g.C;
        float *P = static_cast<float *>(ws);
        const int nblk = cdiv(Mo, 32);
        const dim3 grid(std::max(1, std::min(cdiv(nblk, kThreads / 64), 4 * kNumCUs)));
        if (p.njb == 1)
            hipLaunchKernelGGL((qconv_bwd_data_cols_kernel<T, 1>), grid, dim3(kThreads), p.smem, st,
                               static_cast<const T *>(gy), static_cast<const T *>(ta), static_cast<const T *>(tb),
                               static_cast<const T *>(wa), static_cast<const T *>(wb), static_cast<const T *>(wc), P,
                               (int)Mo, g.O, g.C, J);
        else
            hipLaunchKernelGGL((qconv_bwd_data_cols_kernel<T, 2>), grid, dim3(kThreads), p.smem, st,
                               static_cast<const T *>(gy), static_cast<const T *>(ta), static_cast<const T *>(tb),
                               static_cast<const T *>(wa), static_cast<const T *>(wb), static_cast<const T *>(wc), P,
                               (int)Mo, g.O, g.C, J);
        const ql_status s0 = hip_status();
        if (s0 != QL_OK) return s0;
        const long long M = (long long)g.N * g.H * g.W;
        hipLaunchKernelGGL((qconv_bwd_data_col2im_kernel<T>), dim3(grid_1d(M)), dim3(kThreads), 0, st, P,
                           static_cast<T *>(dx), g.N, g.H, g.W, g.C, g.KH, g.KW, g.SH, g.SW, g.PH, g.PW, g.HO, g.WO);
        return hip_status();
    }
    const int khkw = g.KH * g.KW;
    BwdDataArgs a{};
    ql_status s = QL_OK;
    if (p.natw) {
        a.wt[0] = wa; a.wt[1] = wb; a.wt[2] = wc;
    } else {
        T *wt = static_cast<T *>(ws);
        hipLaunchKernelGGL((qconv_weight_transpose_kernel<T>), dim3(cdiv(g.C, 32), cdiv(g.O, 32), g.terms() * khkw),
                           dim3(kThreads), 0, st, static_cast<const T *>(wa), static_cast<const T *>(wb),
                           static_cast<const T *>(wc), wt, g.O, khkw, g.C);
        s = hip_status();
        if (s != QL_OK) return s;
        const size_t wsz = (size_t)g.O * khkw * g.C;
        a.wt[0] = wt; a.wt[1] = wt + wsz; a.wt[2] = wt + 2 * wsz;
    }
    a.gy = gy; a.ta = ta; a.tb = tb;
    a.dx = dx;
    a.ws = reinterpret_cast<float *>(static_cast<char *>(ws) + p.wt_bytes);
    a.zero = zero_page();
    if (!a.zero) return QL_EHIP;
    a.N = g.N; a.H = g.H; a.W = g.W; a.C = g.C; a.O = g.O; a.KH = g.KH; a.KW = g.KW;
    a.SH = g.SH; a.SW = g.SW; a.PH = g.PH; a.PW = g.PW; a.HO = g.HO; a.WO = g.WO;
    a.M = g.N * g.H * g.W;
    a.K = khkw * g.O;
    a.row_tiles = p.row_tiles; a.col_tiles = p.col_tiles;
    a.splits = p.splits; a.stages_per_split = p.sps; a.stages_total = p.stages_total;
    a.fd_hw = make_fastdiv(g.H * g.W);
    a.fd_w = make_fastdiv(g.W);
    a.fd_o = make_fastdiv(g.O);
    a.fd_kw = make_fastdiv(g.KW);
    a.fd_sh = make_fastdiv(g.SH);
    a.fd_sw = make_fastdiv(g.SW);
    a.neuron = g.ne;
    a.xin = xin;
    a.pm = p.pm ? 1 : 0;
    a.ops = p.KE > 0 ? std::max(1, g.O / p.KE) : 1;  // (the narrow and few-channel plans set no K step)
    a.fd_n = make_fastdiv(g.N);
    a.fd_ops = make_fastdiv(a.ops);
    a.order = p.order;
    if (p.narrow) {
        const dim3 grid((unsigned)(narrow_waves(a.M) / (kThreads / 64)));
#define QL_BD_NARROW(CB, NCH)                                                                                        \
    do {                                                                                                             \
        if (p.s1)                                                                                                    \
            hipLaunchKernelGGL((qconv_bwd_data_narrow_kernel<T, CB, NCH, true>), grid, dim3(kThreads), 0, st, a);  \
        else                                                                                                         \
            hipLaunchKernelGGL((qconv_bwd_data_narrow_kernel<T, CB, NCH, false>), grid, dim3(kThreads), 0, st, a); \
    } while (0)
        switch (p.nch) {
            case 1: QL_BD_NARROW(1, 1); break;
            case 2: QL_BD_NARROW(1, 2); break;
            case 3: QL_BD_NARROW(1, 3); break;
            case 4: QL_BD_NARROW(1, 4); break;
            case 5: QL_BD_NARROW(1, 5); break;
            case 6: QL_BD_NARROW(1, 6); break;
            case 7: QL_BD_NARROW(1, 7); break;
            case 8: QL_BD_NARROW(1, 8); break;
            case 9: QL_BD_NARROW(1, 9); break;
            default: return QL_EINVAL;  // (the planner takes no other shape)
        }
#undef QL_BD_NARROW
        return hip_status();
    }
    const dim3 grid(p.row_tiles * p.col_tiles * p.splits), block(kThreads);
    // channel-aligned K steps (each within one tap): stride 1, natural weight tiles, O a multiple of KE
    const bool bd_ca = p.ca;
    const int om = g.om();
#define QL_BD_PIPE_N(BR, BCOL, WR, WC, NS, NW, OM)                                                                     \
    do {                                                                                                               \
        if (p.s1)                                                                                                      \
            hipLaunchKernelGGL((qconv_bwd_data_kernel<T, BR, BCOL, WR, WC, NS, true, NW, false, OM>), grid, block, 0, st, \
                               a);                                                                                     \
        else                                                                                                           \
            hipLaunchKernelGGL((qconv_bwd_data_kernel<T, BR, BCOL, WR, WC, NS, false, NW, false, OM>), grid, block, 0,  \
                               st, a);                                                                                 \
    } while (0)
#define QL_BD_PIPE_OM(BR, BCOL, WR, WC, NS, OM)                                                                        \
    do {                                                                                                               \
        if constexpr (sizeof(T) == 2) {                                                                                \
            if (bd_ca) {                                                                                               \
                hipLaunchKernelGGL((qconv_bwd_data_kernel<T, BR, BCOL, WR, WC, NS, true, true, true, OM>), grid, block, \
                                   0, st, a);                                                                          \
                break;                                                                                                 \
            }                                                                                                          \
            if (p.natw) {                                                                                              \
                QL_BD_PIPE_N(BR, BCOL, WR, WC, NS, true, OM);                                                          \
                break;                                                                                                 \
            }                                                                                                          \
        }                                                                                                              \
        QL_BD_PIPE_N(BR, BCOL, WR, WC, NS, false, OM);                                                                 \
    } while (0)
#define QL_BD_PIPE(BR, BCOL, WR, WC, NS) QL_BD_PIPE_OM(BR, BCOL, WR, WC, NS, OM_QUADRA)
#define QL_BD_GEN_OM(BR, BCOL, OM)                                                                                 \
    do {                                                                                                           \
        if (p.s1)                                                                                                  \
            hipLaunchKernelGGL((qconv_bwd_data_generic_kernel<T, BR, BCOL, 2, 2, 64, false, true, OM>), grid, block, \
                               0, st, a);                                                                          \
        else                                                                                                       \
            hipLaunchKernelGGL((qconv_bwd_data_generic_kernel<T, BR, BCOL, 2, 2, 64, false, false, OM>), grid,      \
                               block, 0, st, a);                                                                   \
    } while (0)
#define QL_BD_GEN(BR, BCOL) QL_BD_GEN_OM(BR, BCOL, OM_QUADRA)
#define QL_BD_VARIANT(OM)                                                                                          \
    do {                                                                                                           \
        if (!p.veck)                                                                                               \
            QL_BD_GEN_OM(64, 128, OM);                                                                             \
        else if (p.cfg == 3)                                                                                       \
            QL_BD_PIPE_OM(128, 128, 1, 4, 3, OM);                                                                  \
        else                                                                                                       \
            QL_BD_PIPE_OM(64, 128, 1, 4, 4, OM);                                                                   \
    } while (0)
    if (om == OM_PAIR) {
        QL_BD_VARIANT(OM_PAIR);
    } else if (om == OM_SQUARE) {
        QL_BD_VARIANT(OM_SQUARE);
    } else if (om == OM_SQIN) {
        QL_BD_VARIANT(OM_SQIN);
    } else if (om == OM_QSQ) {
        QL_BD_VARIANT(OM_QSQ);
    } else if (p.veck && p.cfg == 4) {
        if constexpr (sizeof(T) == 2)
            hipLaunchKernelGGL((qconv_bwd_data_wide_kernel<256, 256, 2, 4, 3>), grid, dim3(512), 0, st, a);
    } else if (p.veck) {
        if (p.cfg == 0)
            QL_BD_PIPE(128, 128, 2, 2, 3);
        else if (p.cfg == 1)
            QL_BD_PIPE(64, 128, 2, 2, 4);
        else if (p.cfg == 3)
            QL_BD_PIPE(128, 128, 1, 4, 3);
        else if (p.cfg == 5)
            QL_BD_PIPE(64, 128, 1, 4, 4);
        else
            QL_BD_PIPE(128, 64, 2, 2, 4);
    } else if (p.cfg == 0) {
        QL_BD_GEN(128, 128);
    } else {
        QL_BD_GEN(64, 128);
    }
#undef QL_BD_VARIANT
#undef QL_BD_PIPE
#undef QL_BD_PIPE_OM
#undef QL_BD_PIPE_N
#undef QL_BD_GEN
#undef QL_BD_GEN_OM
    s = hip_status();
    if (s != QL_OK || p.splits == 1) return s;
    const long long total = (long long)a.M * g.C;
    // the neuron type's last step on the summed partials: + G (T4 + identity), x 2 X (T2);
    // (T2&4's partials already include their 2 X o (c term))
    const int mode = g.ne == NEURON_T4I ? 1 : (g.ne == NEURON_T2 ? 2 : 0);
    const T *src = static_cast<const T *>(mode == 1 ? gy : (mode == 2 ? xin : nullptr));
    if (g.C % 4 == 0)
        hipLaunchKernelGGL((qconv_sum_splits_kernel<T, true>), dim3(grid_1d(total / 4)), dim3(kThreads), 0, st,
                           static_cast<const float *>(a.ws), p.splits, total, static_cast<T *>(dx), mode, src);
    else
        hipLaunchKernelGGL((qconv_sum_splits_kernel<T, false>), dim3(grid_1d(total)), dim3(kThreads), 0, st,
                           static_cast<const float *>(a.ws), p.splits, total, static_cast<T *>(dx), mode, src);
    return hip_status();
}


ql_status run_bwd_data(const Geom &g, const BwdDataPlan &p, const void *gy, const void *ta, const void *tb,
                       const void *xin, const void *wa, const void *wb, const void *wc, void *dx, void *ws,
                       hipStream_t st) {
    return g.dt == QL_BF16 ? launch_bwd_data<uint16_t>(g, p, gy, ta, tb, xin, wa, wb, wc, dx, ws, st)
                           : launch_bwd_data<float>(g, p, gy, ta, tb, xin, wa, wb, wc, dx, ws, st);
}

}  // namespace host
}  // namespace ql
