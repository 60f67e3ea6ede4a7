// qlaunch_fwd.hip -- launches of the forward kernels (pipelined, few-channel, generic, split-K combine).
#include "qhost.h"
#include "qconv_fwd.h"
#include "qconv_fwd_smallc.h"
#include "qconv_generic.h"

namespace ql {
namespace host {

template <typename T>
ql_status launch_fwd(const Geom &g, const FwdPlan &p, const void *x, const void *wa, const void *wb, const void *wc,
                     const float *ba, const float *bb, const float *bc, void *y, void *ta, void *tb, void *ws,
                     const EpiArgs &epi, float *stat_part, hipStream_t st) {
    FwdArgs a{};
    a.epi = epi;
    a.stat_part = stat_part;  // (set by the caller only where the kernel's staged epilogue runs)
    if (p.smallc) {
        a.x = x;
        a.w[0] = wa; a.w[1] = wb; a.w[2] = wc;
        a.bias[0] = ba; a.bias[1] = bb; a.bias[2] = bc;
        a.y = y; a.ta = ta; a.tb = tb;
        a.N = g.N; a.H = g.H; a.W = g.W; a.C = g.C; a.O = g.O; a.KH = g.KH; a.KW = g.KW;
        a.SH = g.SH; a.SW = g.SW; a.PH = g.PH; a.PW = g.PW; a.HO = g.HO; a.WO = g.WO;
        a.M = g.N * g.HO * g.WO;
        a.K = g.KH * g.KW * g.C;
        a.splits = 1;
        a.fd_howo = make_fastdiv(g.HO * g.WO);
        a.fd_wo = make_fastdiv(g.WO);
        a.fd_c = make_fastdiv(g.C);
        a.fd_kw = make_fastdiv(g.KW);
        a.neuron = g.ne;
        const bool ep = epi.scale || epi.shift || epi.relu;
        // groups of 32 pixels per wave (the next group's loads overlap the current one's stores)
        const long long groups = cdiv(a.M, 32);
        const int gpw = std::max(1, env_override("QLAYER_FWD_SMALLC_GPW", 2));
        const dim3 grid((unsigned)std::max<long long>(
            1, std::min<long long>(cdiv(groups, (long long)(kThreads / 64) * gpw), 4 * kNumCUs)));
#define QL_FWD_SMALLC(OB)                                                                              \
    do {                                                                                               \
        if (ep)                                                                                        \
            hipLaunchKernelGGL((qconv_fwd_smallc_kernel<T, OB, true>), grid, dim3(kThreads), 0, st, a);  \
        else                                                                                           \
            hipLaunchKernelGGL((qconv_fwd_smallc_kernel<T, OB, false>), grid, dim3(kThreads), 0, st, a); \
    } while (0)
        if (g.O == 64) QL_FWD_SMALLC(2);
        else QL_FWD_SMALLC(1);
#undef QL_FWD_SMALLC
        return hip_status();
    }
    a.x = x;
    a.w[0] = wa; a.w[1] = wb; a.w[2] = wc;
    char *wsb = static_cast<char *>(ws);
    if (p.pad) {
        // Zero-pad X and the three weights to Cp channels in the workspace.
        PadSegments sg{};
        const void *srcs[4] = {x, wa, wb, wc};
        const long long wrows = (long long)g.O * g.KH * g.KW;
        const long long rows[4] = {(long long)g.N * g.H * g.W, wrows, g.terms() >= 2 ? wrows : 0,
                                   g.terms() >= 3 ? wrows : 0};  // (terms the type lacks: nothing to pad)
        for (int i = 0; i < 4; ++i) {
            sg.src[i] = srcs[i];
            sg.dst[i] = wsb + (i == 0 ? 0 : p.xpad_bytes + (size_t)(i - 1) * p.wpad_bytes);
            sg.rows[i] = rows[i];
        }
        // (one thread per row when a padded row is one 16-byte vector, else per element)
        const long long pad_items = rows[0] * (p.Cp * (int)sizeof(T) == 16 ? 1 : p.Cp);
        hipLaunchKernelGGL((qconv_pad_channels_kernel<T, 4>), dim3(grid_1d(pad_items), 4), dim3(kThreads), 0, st,
                           sg, g.C, p.Cp);
        const ql_status s0 = hip_status();
        if (s0 != QL_OK) return s0;
        a.x = sg.dst[0];
        a.w[0] = sg.dst[1]; a.w[1] = sg.dst[2]; a.w[2] = sg.dst[3];
    }
    const int C = p.Cp;  // channels the GEMM sees
    a.bias[0] = ba; a.bias[1] = bb; a.bias[2] = bc;
    a.y = y; a.ta = ta; a.tb = tb;
    a.ws = reinterpret_cast<float *>(wsb + p.xpad_bytes + 3 * p.wpad_bytes);
    a.zero = zero_page();
    if (!a.zero) return QL_EHIP;
    a.N = g.N; a.H = g.H; a.W = g.W; a.C = C; a.O = g.O; a.KH = g.KH; a.KW = g.KW;
    a.SH = g.SH; a.SW = g.SW; a.PH = g.PH; a.PW = g.PW; a.HO = g.HO; a.WO = g.WO;
    a.M = g.N * g.HO * g.WO;
    a.K = g.KH * g.KW * C;
    a.row_tiles = p.row_tiles; a.col_tiles = p.col_tiles;
    a.splits = p.splits; a.stages_per_split = p.sps; a.stages_total = p.stages_total;
    a.fd_howo = make_fastdiv(g.HO * g.WO);
    a.fd_wo = make_fastdiv(g.WO);
    a.fd_c = make_fastdiv(C);
    a.fd_kw = make_fastdiv(g.KW);
    a.pm = p.pm ? 1 : 0;
    a.cps = C / p.KE;
    a.fd_n = make_fastdiv(g.N);
    a.fd_cps = make_fastdiv(std::max(1, a.cps));
    a.neuron = g.ne;
    if (p.narrow) {
        const dim3 grid((unsigned)(narrow_waves(a.M) / (kThreads / 64)));
        const bool ep = epi.scale || epi.shift || epi.relu || stat_part != nullptr;
#define QL_FWD_NARROW(OB, NCH)                                                                                  \
    do {                                                                                                        \
        if (ep)                                                                                                 \
            hipLaunchKernelGGL((qconv_fwd_narrow_kernel<T, OB, NCH, true>), grid, dim3(kThreads), 0, st, a);  \
        else                                                                                                    \
            hipLaunchKernelGGL((qconv_fwd_narrow_kernel<T, OB, NCH, false>), grid, dim3(kThreads), 0, st, a); \
    } while (0)
        switch (p.nch) {
            case 1: QL_FWD_NARROW(1, 1); break;
            case 2: QL_FWD_NARROW(1, 2); break;
            case 3: QL_FWD_NARROW(1, 3); break;
            case 4: QL_FWD_NARROW(1, 4); break;
            case 5: QL_FWD_NARROW(1, 5); break;
            case 6: QL_FWD_NARROW(1, 6); break;
            case 7: QL_FWD_NARROW(1, 7); break;
            case 8: QL_FWD_NARROW(1, 8); break;
            case 9: QL_FWD_NARROW(1, 9); break;
            default: return QL_EINVAL;  // (the planner takes no other shape)
        }
#undef QL_FWD_NARROW
        return hip_status();
    }
    if (p.ksplit) return launch_fwd_ksplit<T>(p, a, epi.scale || epi.shift || epi.relu || stat_part != nullptr, st);
    if (p.xsq_bytes) {
        // T2: X o X once, instead of squaring every fragment in the MFMA loop
        T *xsq = reinterpret_cast<T *>(wsb + p.xpad_bytes + 3 * p.wpad_bytes + p.part_bytes);
        const long long n = (long long)g.N * g.H * g.W * C;
        hipLaunchKernelGGL((qconv_square_kernel<T>), dim3(grid_1d(n / g.vec())), dim3(kThreads), 0, st,
                           static_cast<const T *>(a.x), xsq, n);
        const ql_status s0 = hip_status();
        if (s0 != QL_OK) return s0;
        a.x = xsq;
        a.xsq = 1;
    }
    const dim3 grid(p.row_tiles * p.col_tiles * p.splits), block(kThreads);
    const int om = g.om();
    if (p.veck && om != OM_QUADRA) {
        const bool ca = p.ca;
#define QL_FWD_OM(OM)                                                                                          \
    do {                                                                                                        \
        if (ca)                                                                                                 \
            hipLaunchKernelGGL((qconv_fwd_kernel<T, 64, 128, 2, 2, 4, true, 256, OM>), grid, block, 0, st, a);  \
        else                                                                                                    \
            hipLaunchKernelGGL((qconv_fwd_kernel<T, 64, 128, 2, 2, 4, false, 256, OM>), grid, block, 0, st, a); \
    } while (0)
        if (om == OM_PAIR) QL_FWD_OM(OM_PAIR);
        else if (om == OM_SQUARE) QL_FWD_OM(OM_SQUARE);
        else if (om == OM_QSQ) QL_FWD_OM(OM_QSQ);
        else QL_FWD_OM(OM_SQIN);
#undef QL_FWD_OM
    } else if (!p.veck && om != OM_QUADRA) {
        if (om == OM_PAIR)
            hipLaunchKernelGGL((qconv_fwd_generic_kernel<T, 64, 128, 2, 2, 64, false, OM_PAIR>), grid, block, 0, st, a);
        else if (om == OM_SQUARE)
            hipLaunchKernelGGL((qconv_fwd_generic_kernel<T, 64, 128, 2, 2, 64, false, OM_SQUARE>), grid, block, 0, st,
                               a);
        else if (om == OM_QSQ)
            hipLaunchKernelGGL((qconv_fwd_generic_kernel<T, 64, 128, 2, 2, 64, false, OM_QSQ>), grid, block, 0, st, a);
        else
            hipLaunchKernelGGL((qconv_fwd_generic_kernel<T, 64, 128, 2, 2, 64, false, OM_SQIN>), grid, block, 0, st, a);
    } else if (p.veck) {
        // channel-aligned K steps: every step within one tap
        const bool ca = p.ca;
#define QL_FWD(BR, BC, WR, WC, NS, NT)                                                                           \
    do {                                                                                                          \
        if (ca)                                                                                                   \
            hipLaunchKernelGGL((qconv_fwd_kernel<T, BR, BC, WR, WC, NS, true, NT>), grid, dim3(NT), 0, st, a);   \
        else                                                                                                      \
            hipLaunchKernelGGL((qconv_fwd_kernel<T, BR, BC, WR, WC, NS, false, NT>), grid, dim3(NT), 0, st, a);  \
    } while (0)
        switch (p.cfg) {
            case 0: QL_FWD(128, 128, 4, 1, 4, 256); break;
            case 1: QL_FWD(64, 256, 2, 2, 4, 256); break;
            case 2: QL_FWD(128, 128, 2, 2, 4, 256); break;
            case 4: QL_FWD(128, 256, 4, 2, 3, 512); break;
            case 5: QL_FWD(128, 256, 2, 4, 3, 512); break;
            case 6: QL_FWD(128, 256, 4, 2, 4, 512); break;
            default: QL_FWD(64, 128, 2, 2, 4, 256); break;
        }
#undef QL_FWD
    } else if (p.cfg == 0) {
        hipLaunchKernelGGL((qconv_fwd_generic_kernel<T, 128, 128, 2, 2, 64, false>), grid, block, 0, st, a);
    } else {
        hipLaunchKernelGGL((qconv_fwd_generic_kernel<T, 64, 128, 2, 2, 64, false>), grid, block, 0, st, a);
    }
    ql_status s = hip_status();
    if (s != QL_OK || p.splits == 1) return s;
    const long long MO = (long long)a.M * g.O;
    if (g.O % 4 == 0)
        hipLaunchKernelGGL((qconv_fwd_combine_kernel<T, true>), dim3(grid_1d(MO / 4)), dim3(kThreads), 0, st,
                           static_cast<const float *>(a.ws), p.splits, MO, g.O, ba, bb, bc, static_cast<T *>(y),
                           static_cast<T *>(ta), static_cast<T *>(tb), g.ne, static_cast<const T *>(x), epi);
    else
        hipLaunchKernelGGL((qconv_fwd_combine_kernel<T, false>), dim3(grid_1d(MO)), dim3(kThreads), 0, st,
                           static_cast<const float *>(a.ws), p.splits, MO, g.O, ba, bb, bc, static_cast<T *>(y),
                           static_cast<T *>(ta), static_cast<T *>(tb), g.ne, static_cast<const T *>(x), epi);
    return hip_status();
}


ql_status run_fwd(const Geom &g, const FwdPlan &p, const void *x, const void *wa, const void *wb, const void *wc,
                  const float *ba, const float *bb, const float *bc, void *y, void *ta, void *tb, void *ws,
                  const EpiArgs &epi, float *stat_part, hipStream_t st) {
    return g.dt == QL_BF16 ? launch_fwd<uint16_t>(g, p, x, wa, wb, wc, ba, bb, bc, y, ta, tb, ws, epi, stat_part, st)
                           : launch_fwd<float>(g, p, x, wa, wb, wc, ba, bb, bc, y, ta, tb, ws, epi, stat_part, st);
}

}  // namespace host
}  // namespace ql
