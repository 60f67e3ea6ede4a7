// qlaunch_dw.hip -- launches of the depthwise kernels (3 x 3 column kernels, generic kernels, split reduction).
#include "qhost.h"

namespace ql {
namespace host {

// 3 x 3 kernels of one operand mode and channel vector.
template <typename T, int OM, int V, bool VEC>
void dw_launch_k(const DwPlan &p, int pass, int S, const DwArgs &a, dim3 grid, size_t smem, hipStream_t st) {
    if (pass == 0) {
        if constexpr (V == 4) {
            if (S == 1) hipLaunchKernelGGL((qconv_dw_fwd_col_kernel<T, OM, V, VEC, 3, 1, kDwRowsFwd, true>), grid, dim3(kThreads), smem, st, a);
            else hipLaunchKernelGGL((qconv_dw_fwd_col_kernel<T, OM, V, VEC, 3, 2, kDwRowsFwd, true>), grid, dim3(kThreads), smem, st, a);
        }
    } else if (pass == 1) {
        // prefetching the next column fits the registers with bf16 only
        constexpr bool PF = sizeof(T) == 2 && V == 4;
        if (!p.col) hipLaunchKernelGGL((qconv_dw_bwd_data_k_kernel<T, OM, V, VEC, 3, 2>), grid, dim3(kThreads), smem, st, a);
        else if constexpr (V == 4) hipLaunchKernelGGL((qconv_dw_bwd_data_col_kernel<T, OM, V, VEC, 3, kDwRowsBd, PF>), grid, dim3(kThreads), smem, st, a);
    } else if constexpr (V == 4) {
        if (S == 1) hipLaunchKernelGGL((qconv_dw_bwd_weight_col_kernel<T, OM, V, VEC, 3, 1, kDwRowsBw>), grid, dim3(kThreads), 0, st, a);
        else hipLaunchKernelGGL((qconv_dw_bwd_weight_col_kernel<T, OM, V, VEC, 3, 2, kDwRowsBw>), grid, dim3(kThreads), 0, st, a);
    }
}
template <typename T, int OM>
void dw_launch_om(const DwPlan &p, int pass, int S, const DwArgs &a, dim3 grid, size_t smem, hipStream_t st) {
    if constexpr (sizeof(T) == 2) {
        if (p.V == 8) return dw_launch_k<T, OM, 8, true>(p, pass, S, a, grid, smem, st);
    }
    if (p.vec) dw_launch_k<T, OM, 4, true>(p, pass, S, a, grid, smem, st);
    else dw_launch_k<T, OM, 4, false>(p, pass, S, a, grid, smem, st);
}
template <typename T>
void dw_launch_fast(const Geom &g, const DwPlan &p, int pass, const DwArgs &a, dim3 grid, size_t smem,
                    hipStream_t st) {
    switch (g.om()) {
        case OM_QUADRA: dw_launch_om<T, OM_QUADRA>(p, pass, g.SH, a, grid, smem, st); break;
        case OM_PAIR: dw_launch_om<T, OM_PAIR>(p, pass, g.SH, a, grid, smem, st); break;
        case OM_SQUARE: dw_launch_om<T, OM_SQUARE>(p, pass, g.SH, a, grid, smem, st); break;
        default: dw_launch_om<T, OM_SQIN>(p, pass, g.SH, a, grid, smem, st); break;
    }
}

// generic kernels: dispatch a template over (T, OM, V4)
#define QL_DW_DISPATCH(KERNEL, EXTRA, GRID, SMEM)                                                              \
    do {                                                                                                       \
        const bool v4 = g.C % 4 == 0;                                                                          \
        const int om = g.om();                                                                                 \
        if (om == OM_QUADRA) {                                                                                 \
            if (v4) hipLaunchKernelGGL((KERNEL<T, OM_QUADRA, true EXTRA>), GRID, dim3(kThreads), SMEM, st, a);    \
            else hipLaunchKernelGGL((KERNEL<T, OM_QUADRA, false EXTRA>), GRID, dim3(kThreads), SMEM, st, a);      \
        } else if (om == OM_PAIR) {                                                                            \
            if (v4) hipLaunchKernelGGL((KERNEL<T, OM_PAIR, true EXTRA>), GRID, dim3(kThreads), SMEM, st, a);      \
            else hipLaunchKernelGGL((KERNEL<T, OM_PAIR, false EXTRA>), GRID, dim3(kThreads), SMEM, st, a);        \
        } else if (om == OM_SQUARE) {                                                                          \
            if (v4) hipLaunchKernelGGL((KERNEL<T, OM_SQUARE, true EXTRA>), GRID, dim3(kThreads), SMEM, st, a);    \
            else hipLaunchKernelGGL((KERNEL<T, OM_SQUARE, false EXTRA>), GRID, dim3(kThreads), SMEM, st, a);      \
        } else {                                                                                               \
            if (v4) hipLaunchKernelGGL((KERNEL<T, OM_SQIN, true EXTRA>), GRID, dim3(kThreads), SMEM, st, a);      \
            else hipLaunchKernelGGL((KERNEL<T, OM_SQIN, false EXTRA>), GRID, dim3(kThreads), SMEM, st, a);        \
        }                                                                                                      \
    } while (0)
#define QL_NOEXTRA
#define QL_TAPS9 , 9

template <typename T>
ql_status launch_dw_fwd(const Geom &g, const void *x, const void *const *w, const float *const *b, void *y,
                        void *ta, void *tb, const EpiArgs &epi, hipStream_t st) {
    const DwPlan p = plan_dw(g, 0);
    DwArgs a = dw_args(g, p);
    a.epi = epi;
    a.x = x;
    for (int t = 0; t < 3; ++t) { a.w[t] = w[t]; a.bias[t] = b[t]; }
    a.y = y; a.yta = ta; a.ytb = tb;
    if (p.fast) {
        a.zero = zero_page();
        if (!a.zero) return QL_EHIP;
        a.M = (int)p.items;
        const size_t smem = (size_t)g.terms() * (9 + 1) * p.lanes * p.V * sizeof(float);  // filters, biases
        dw_launch_fast<T>(g, p, 0, a, dim3(p.grid), smem, st);
        return hip_status();
    }
    a.M = g.N * g.HO * g.WO;
    const dim3 grid(std::max(1, std::min(cdiv(a.M, kDwPL), cdiv(16 * kNumCUs, p.ct))), p.ct);
    const size_t smem = (size_t)g.terms() * g.KH * g.KW * kDwCB * sizeof(float);
    QL_DW_DISPATCH(qconv_dw_fwd_kernel, QL_NOEXTRA, grid, smem);
    return hip_status();
}

template <typename T>
ql_status launch_dw_bwd_data(const Geom &g, const void *gy, const void *ta, const void *tb, const void *const *w,
                             void *dx, hipStream_t st) {
    const DwPlan p = plan_dw(g, 1);
    DwArgs a = dw_args(g, p);
    a.gy = gy; a.ta = ta; a.tb = tb;
    for (int t = 0; t < 3; ++t) a.w[t] = w[t];
    a.dx = dx;
    if (p.fast) {
        a.zero = zero_page();
        if (!a.zero) return QL_EHIP;
        a.M = (int)p.items;
        const size_t smem = (size_t)g.terms() * 9 * p.lanes * p.V * sizeof(float);
        dw_launch_fast<T>(g, p, 1, a, dim3(p.grid), smem, st);
        return hip_status();
    }
    a.M = g.N * g.H * g.W;
    const dim3 grid(std::max(1, std::min(cdiv(a.M, kDwPL), cdiv(16 * kNumCUs, p.ct))), p.ct);
    const size_t smem = (size_t)g.terms() * g.KH * g.KW * kDwCB * sizeof(float);
    QL_DW_DISPATCH(qconv_dw_bwd_data_kernel, QL_NOEXTRA, grid, smem);
    return hip_status();
}

template <typename T>
ql_status launch_dw_bwd_weight(const Geom &g, const DwPlan &p, const void *x, const void *gy, const void *ta,
                               const void *tb, float *const *dw, float *const *db, void *ws, hipStream_t st) {
    DwArgs a = dw_args(g, p);
    a.x = x; a.gy = gy; a.ta = ta; a.tb = tb;
    for (int t = 0; t < 3; ++t) { a.dw[t] = dw[t]; a.db[t] = db[t]; }
    a.ws = static_cast<float *>(ws);
    a.splits = p.splits;
    a.px_per_split = p.pps;
    a.M = (int)p.items;
    if (p.fast) {
        a.zero = zero_page();
        if (!a.zero) return QL_EHIP;
        dw_launch_fast<T>(g, p, 2, a, dim3(p.splits, p.tiles), 0, st);
    } else {
        const dim3 grid(p.splits, p.ct, p.tg);
        QL_DW_DISPATCH(qconv_dw_bwd_weight_kernel, QL_TAPS9, grid, 0);
    }
    ql_status s = hip_status();
    if (s != QL_OK || p.splits == 1) return s;
    const int taps = g.KH * g.KW, nt = g.terms();
    const int jn = nt * g.C * taps + (db[0] ? nt * g.C : 0);
    hipLaunchKernelGGL(qconv_dw_reduce_kernel<>, dim3(cdiv(jn, 16)), dim3(kThreads), 0, st, a.ws, p.splits, a.J, g.C,
                       taps, nt, dw[0], dw[1], dw[2], db[0], db[1], db[2], db[0] != nullptr);
    return hip_status();
}
#undef QL_DW_DISPATCH
#undef QL_NOEXTRA
#undef QL_TAPS9


ql_status run_dw_fwd(const Geom &g, const void *x, const void *const *w, const float *const *b, void *y, void *ta,
                     void *tb, const EpiArgs &epi, hipStream_t st) {
    return g.dt == QL_BF16 ? launch_dw_fwd<uint16_t>(g, x, w, b, y, ta, tb, epi, st)
                           : launch_dw_fwd<float>(g, x, w, b, y, ta, tb, epi, st);
}
ql_status run_dw_bwd_data(const Geom &g, const void *gy, const void *ta, const void *tb, const void *const *w,
                          void *dx, hipStream_t st) {
    return g.dt == QL_BF16 ? launch_dw_bwd_data<uint16_t>(g, gy, ta, tb, w, dx, st)
                           : launch_dw_bwd_data<float>(g, gy, ta, tb, w, dx, st);
}
ql_status run_dw_bwd_weight(const Geom &g, const DwPlan &p, const void *x, const void *gy, const void *ta,
                            const void *tb, float *const *dw, float *const *db, void *ws, hipStream_t st) {
    return g.dt == QL_BF16 ? launch_dw_bwd_weight<uint16_t>(g, p, x, gy, ta, tb, dw, db, ws, st)
                           : launch_dw_bwd_weight<float>(g, p, x, gy, ta, tb, dw, db, ws, st);
}

}  // namespace host
}  // namespace ql
