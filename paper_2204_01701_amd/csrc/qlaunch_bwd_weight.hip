// qlaunch_bwd_weight.hip -- launches of the weight-gradient kernels (pipelined, generic, split reduction).
#include "qhost.h"
#include "qconv_bwd_weight.h"
#include "qconv_bwd_weight16.h"
#include "qconv_bwd_weight_narrow.h"
#include "qconv_generic.h"

namespace ql {
namespace host {

// The weight-gradient split reduction: dW_t and db_t from the partials
// [split][3][O KH KW C] and [split][3][O], summed in split order.
ql_status reduce_bw_partials(const Geom &g, int splits, const BwdWeightArgs &a, float *dwa, float *dwb, float *dwc,
                             float *dba, float *dbb, float *dbc, hipStream_t st) {
    const long long ndw = (long long)g.O * g.KH * g.KW * g.C;  // dW_t as stored
    if (3 * ndw < (1LL << 20) && splits >= 16 && ndw % 4 == 0)
        hipLaunchKernelGGL(qconv_bwd_weight_reduce2dv_kernel<>, dim3(grid_1d((3 * ndw / 4 + 3 * g.O) * 16)),
                           dim3(kThreads), 0, st, static_cast<const float *>(a.ws_dw),
                           static_cast<const float *>(a.ws_db), splits, ndw, g.O, dwa, dwb, dwc, dba, dbb, dbc,
                           a.want_db, g.terms());
    else if (3 * ndw < (1LL << 20) && splits >= 16)
        hipLaunchKernelGGL((qconv_bwd_weight_reduce2d_kernel<16>), dim3(grid_1d((3 * ndw + 3 * g.O) * 16)),
                           dim3(kThreads), 0, st, static_cast<const float *>(a.ws_dw),
                           static_cast<const float *>(a.ws_db), splits, ndw, g.O, dwa, dwb, dwc, dba, dbb, dbc,
                           a.want_db, g.terms());
    else if (ndw % 4 == 0)
        hipLaunchKernelGGL((qconv_bwd_weight_reduce_kernel<true>), dim3(grid_1d(3 * ndw / 4 + 3 * g.O)),
                           dim3(kThreads), 0, st, static_cast<const float *>(a.ws_dw),
                           static_cast<const float *>(a.ws_db), splits, ndw, g.O, dwa, dwb, dwc, dba, dbb, dbc,
                           a.want_db, g.terms());
    else
        hipLaunchKernelGGL((qconv_bwd_weight_reduce_kernel<false>), dim3(grid_1d(3 * ndw + 3 * g.O)),
                           dim3(kThreads), 0, st, static_cast<const float *>(a.ws_dw),
                           static_cast<const float *>(a.ws_db), splits, ndw, g.O, dwa, dwb, dwc, dba, dbb, dbc,
                           a.want_db, g.terms());
    return hip_status();
}

template <typename T>
ql_status launch_bwd_weight(const Geom &g, const BwdWeightPlan &p, const void *x, const void *gy, const void *ta,
                            const void *tb, float *dwa, float *dwb, float *dwc, float *dba, float *dbb, float *dbc,
                            void *ws, hipStream_t st) {
    BwdWeightArgs a{};
    a.x = x; a.gy = gy; a.ta = ta; a.tb = tb;
    char *wsb = static_cast<char *>(ws);
    if (p.pad) {
        // Zero-pad X to Cp channels in the workspace; dW_t is stored with the true C.
        PadSegments sg{};
        sg.src[0] = x;
        sg.dst[0] = wsb;
        sg.rows[0] = (long long)g.N * g.H * g.W;
        const long long pad_items = sg.rows[0] * (p.Cp * (int)sizeof(T) == 16 ? 1 : p.Cp);
        hipLaunchKernelGGL((qconv_pad_channels_kernel<T, 1>), dim3(grid_1d(pad_items), 1), dim3(kThreads), 0, st,
                           sg, g.C, p.Cp);
        const ql_status s0 = hip_status();
        if (s0 != QL_OK) return s0;
        a.x = wsb;
    }
    const int C = p.Cp;  // channels the GEMM sees
    a.dw[0] = dwa; a.dw[1] = dwb; a.dw[2] = dwc;
    a.db[0] = dba; a.db[1] = dbb; a.db[2] = dbc;
    a.ws_dw = reinterpret_cast<float *>(wsb + p.xpad_bytes);
    a.ws_db = reinterpret_cast<float *>(wsb + p.xpad_bytes + p.dw_bytes);
    a.zero = zero_page();
    if (!a.zero) return QL_EHIP;
    a.N = g.N; a.H = g.H; a.W = g.W; a.C = C; a.O = g.O; a.KH = g.KH; a.KW = g.KW;
    a.SH = g.SH; a.SW = g.SW; a.PH = g.PH; a.PW = g.PW; a.HO = g.HO; a.WO = g.WO;
    a.M = g.N * g.HO * g.WO;
    a.KP = g.KH * g.KW * C;
    a.C_out = g.C;
    a.row_tiles = p.row_tiles; a.col_tiles = p.col_tiles;
    a.splits = p.splits; a.stages_per_split = p.sps; a.stages_total = p.stages_total;
    a.want_db = dba != nullptr;
    a.fd_howo = make_fastdiv(g.HO * g.WO);
    a.fd_wo = make_fastdiv(g.WO);
    a.fd_c = make_fastdiv(C);
    a.fd_kw = make_fastdiv(g.KW);
    a.lin = g.SH == 1 && g.SW == 1 && g.HO == g.H && g.WO == g.W && env_override("QLAYER_BWD_WEIGHT_LIN", 1) != 0;
    a.lin_dq = (p.KE / g.WO) % g.HO;
    a.lin_dr = p.KE % g.WO;
    a.neuron = g.ne;
    if (p.narrow) {
#define QL_BW_NARROW(NF) \
    hipLaunchKernelGGL((qconv_bwd_weight_narrow_kernel<T, NF>), dim3(p.splits, p.nob), dim3(kThreads), 0, st, a)
        switch (p.nf) {
            case 1: QL_BW_NARROW(1); break;
            case 2: QL_BW_NARROW(2); break;
            case 3: QL_BW_NARROW(3); break;
            case 4: QL_BW_NARROW(4); break;
            case 5: QL_BW_NARROW(5); break;
            case 6: QL_BW_NARROW(6); break;
            case 7: QL_BW_NARROW(7); break;
            case 8: QL_BW_NARROW(8); break;
            case 9: QL_BW_NARROW(9); break;
            default: return QL_EINVAL;  // (the planner takes no other shape)
        }
#undef QL_BW_NARROW
        const ql_status s = hip_status();
        if (s != QL_OK || p.splits == 1) return s;
        return reduce_bw_partials(g, p.splits, a, dwa, dwb, dwc, dba, dbb, dbc, st);
    }
    const dim3 grid(p.row_tiles * p.col_tiles * p.splits), block(kThreads);
    const int om = g.om();
    if (om != OM_QUADRA) {
        // the other neuron types: the 128 x 64 pipelined tile (bf16) or the generic 128 x 64 kernel
#define QL_BW_OM(OM)                                                                                               \
    do {                                                                                                           \
        if (p.pipe) {                                                                                              \
            if constexpr (sizeof(T) == 2)                                                                          \
                hipLaunchKernelGGL((qconv_bwd_weight_kernel<128, 64, 2, 2, 4, 256, OM>), grid, block, 0, st, a);   \
        } else if (p.veck) {                                                                                       \
            hipLaunchKernelGGL((qconv_bwd_weight_generic_kernel<T, 128, 64, 2, 2, 64, 4, true, OM>), grid, block, 0, \
                               st, a);                                                                             \
        } else {                                                                                                   \
            hipLaunchKernelGGL((qconv_bwd_weight_generic_kernel<T, 128, 64, 2, 2, 64, 4, false, OM>), grid, block,   \
                               0, st, a);                                                                          \
        }                                                                                                          \
    } while (0)
        if (om == OM_PAIR) QL_BW_OM(OM_PAIR);
        else if (om == OM_SQUARE) QL_BW_OM(OM_SQUARE);
        else if (om == OM_QSQ) QL_BW_OM(OM_QSQ);
        else QL_BW_OM(OM_SQIN);
#undef QL_BW_OM
    } else if constexpr (sizeof(T) == 2) {
        if (p.pipe) {
            switch (p.cfg) {
                case 0: hipLaunchKernelGGL((qconv_bwd_weight_kernel<128, 64, 2, 2, 4>), grid, block, 0, st, a); break;
                case 1: hipLaunchKernelGGL((qconv_bwd_weight_kernel<128, 128, 2, 2, 4>), grid, block, 0, st, a); break;
                case 3: hipLaunchKernelGGL((qconv_bwd_weight16_kernel<128, 4>), grid, block, 0, st, a); break;
                case 4:
                    hipLaunchKernelGGL((qconv_bwd_weight16_kernel<128, 4, 2>), grid, dim3(kBwThreads[4]), 0, st, a);
                    break;
                case 5:
                    hipLaunchKernelGGL((qconv_bwd_weight16_kernel<128, 5, 1, 128>), grid, dim3(kBwThreads[5]), 0, st,
                                       a);
                    break;
                default: hipLaunchKernelGGL((qconv_bwd_weight_kernel<64, 64, 2, 2, 4>), grid, block, 0, st, a); break;
            }
        }
    }
    if constexpr (sizeof(T) == 4) {
        if (p.pipe && om == OM_QUADRA) {
            switch (p.cfg) {
                case 4:
                    hipLaunchKernelGGL((qconv_bwd_weight16_kernel<128, 4, 2, 64, float>), grid, dim3(kBwThreads[4]), 0,
                                       st, a);
                    break;
                case 5:
                    hipLaunchKernelGGL((qconv_bwd_weight16_kernel<128, 5, 1, 128, float>), grid, dim3(kBwThreads[5]),
                                       0, st, a);
                    break;
                default:
                    hipLaunchKernelGGL((qconv_bwd_weight16_kernel<128, 4, 1, 64, float>), grid, block, 0, st, a);
                    break;
            }
        }
    }
    if (!p.pipe && om == OM_QUADRA) {
        if (p.veck)
            hipLaunchKernelGGL((qconv_bwd_weight_generic_kernel<T, 128, 64, 2, 2, 64, 4, true>), grid, block, 0, st, a);
        else
            hipLaunchKernelGGL((qconv_bwd_weight_generic_kernel<T, 128, 64, 2, 2, 64, 4, false>), grid, block, 0, st,
                               a);
    }
    ql_status s = hip_status();
    if (s != QL_OK || p.splits == 1) return s;
    return reduce_bw_partials(g, p.splits, a, dwa, dwb, dwc, dba, dbb, dbc, st);
}


ql_status run_bwd_weight(const Geom &g, const BwdWeightPlan &p, const void *x, const void *gy, const void *ta,
                         const void *tb, float *dwa, float *dwb, float *dwc, float *dba, float *dbb, float *dbc,
                         void *ws, hipStream_t st) {
    return g.dt == QL_BF16
               ? launch_bwd_weight<uint16_t>(g, p, x, gy, ta, tb, dwa, dwb, dwc, dba, dbb, dbc, ws, st)
               : launch_bwd_weight<float>(g, p, x, gy, ta, tb, dwa, dwb, dwc, dba, dbb, dbc, ws, st);
}

}  // namespace host
}  // namespace ql
