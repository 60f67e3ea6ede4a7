// qlayer_api.hip -- host side of the C ABI declared in include/qlayer.h:
// argument validation and workspace carving, then the launchers of the
// kernel families (qlaunch_*.hip) on the caller's stream; the forward
// epilogue's statistics kernels.  Nothing here touches tensor data on the
// host and nothing allocates device memory.
#include <mutex>

#include "qhost.h"

namespace ql {
// The 16 zero bytes masked-off lanes of the pipelined kernels load.
__device__ __attribute__((aligned(16))) uint32_t g_zero16[4] = {0u, 0u, 0u, 0u};

namespace host {
// Device address of g_zero16 on the current device, resolved once per device
// (std::call_once: host threads calling concurrently see one resolution).
constexpr int kMaxDevices = 64;
const void *zero_page() {
    static std::once_flag once[kMaxDevices];
    static const void *addr[kMaxDevices] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::call_once(once[dev], [dev] {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(ql::g_zero16)) == hipSuccess) addr[dev] = p;
    });
    return addr[dev];
}
}  // namespace host

// Scratch memory of qlayer_conv2d_bwd_weight_noalloc, the entry point for
// callers that cannot allocate: one array per GPU the library runs on, held
// until the process ends.  Host code never uses its name as an address (on
// the host it is a stand-in symbol): the device address comes from
// hipGetSymbolAddress, once per device.
constexpr size_t kScratchBytes = QLAYER_NOALLOC_SCRATCH_BYTES;
static __device__ __attribute__((aligned(256))) unsigned char scratch[kScratchBytes];

namespace host {
// Device address of `scratch` on the current device (nullptr if it cannot be resolved).
void *scratch_ptr() {
    static std::once_flag once[kMaxDevices];
    static void *addr[kMaxDevices] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::call_once(once[dev], [dev] {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) == hipSuccess) addr[dev] = p;
    });
    return addr[dev];
}
}  // namespace host
}  // namespace ql

using namespace ql;
using namespace ql::host;

namespace {

// The forward epilogue's statistics: partial sums per pixel tile (gathered by
// the staged forward kernel) or per part of rows (a pass over the stored Y'),
// then one reduction in part order.
struct StatPlan {
    bool on, fused;
    int nparts, rpp;  // parts; rows per part of the separate pass
    size_t bytes;
};

StatPlan plan_stats(const Geom &g, const ql_epilogue *e) {
    StatPlan s{};
    s.on = e && e->sum;
    if (!s.on) return s;
    const int M = g.N * g.HO * g.WO;
    FwdPlan p{};
    if (!g.dw) p = plan_fwd(g);
    s.fused = !g.dw && fwd_stats_fused(g, p);
    if (s.fused) {
        s.nparts = p.stat_parts;
    } else {
        s.rpp = std::max(64, cdiv(M, 1024));
        s.nparts = cdiv(M, s.rpp);
    }
    s.bytes = align_up((size_t)s.nparts * 2 * g.O * sizeof(float));
    return s;
}

size_t fwd_ws_bytes(const Geom &g, const ql_epilogue *e) {
    return (g.dw ? 0 : plan_fwd(g).ws_bytes) + plan_stats(g, e).bytes;
}

ql_status fwd_common(const Geom &g, const void *x, const void *wa, const void *wb, const void *wc, const float *ba,
                     const float *bb, const float *bc, void *y, void *ta, void *tb, const ql_epilogue *e, void *ws,
                     size_t ws_bytes, void *stream) {
    const int nt = g.terms();
    // pointers of terms the neuron type lacks are ignored
    if (nt < 3) { wc = nullptr; bc = nullptr; }
    if (nt < 2) { wb = nullptr; bb = nullptr; tb = nullptr; }
    if (g.ne == NEURON_T2) ta = nullptr;  // (nothing is saved: its backward takes X)
    if (!x || !wa || (nt >= 2 && !wb) || (nt >= 3 && !wc)) return QL_EINVAL;
    const bool saved = g.ne == NEURON_T2 ? false : (nt >= 2 ? (ta && tb) : ta != nullptr);
    if (!y && !saved) return QL_EINVAL;
    EpiArgs epi{};
    if (e) {
        // the epilogue transforms Y: it needs Y; the statistics come as a pair
        const bool any = e->scale || e->shift || e->relu || e->sum || e->sumsq;
        if (any && !y) return QL_EINVAL;
        if ((e->sum == nullptr) != (e->sumsq == nullptr)) return QL_EINVAL;
        const void *eps[] = {e->scale, e->shift, e->sum, e->sumsq};
        for (const void *q : eps)
            if (q && !aligned16(q)) return QL_EINVAL;
        epi.scale = e->scale;
        epi.shift = e->shift;
        epi.relu = e->relu != 0;
    }
    const void *ptrs[] = {x, wa, wb, wc, ba, bb, bc, y, ta, tb};
    for (const void *q : ptrs)
        if (q && !aligned16(q)) return QL_EINVAL;
    const StatPlan sp = plan_stats(g, e);
    const size_t main_bytes = g.dw ? 0 : plan_fwd(g).ws_bytes;
    if (ws_bytes < main_bytes + sp.bytes || (main_bytes + sp.bytes && !ws)) return QL_EWORKSPACE;
    if (ws && !aligned16(ws)) return QL_EINVAL;
    float *stat_part = sp.on ? reinterpret_cast<float *>(static_cast<char *>(ws) + main_bytes) : nullptr;
    hipStream_t st = static_cast<hipStream_t>(stream);
    ql_status s;
    if (g.dw) {
        const void *w[3] = {wa, wb, wc};
        const float *b[3] = {ba, bb, bc};
        s = run_dw_fwd(g, x, w, b, y, ta, tb, epi, st);
    } else {
        const FwdPlan p = plan_fwd(g);
        float *fused_part = sp.fused ? stat_part : nullptr;
        s = run_fwd(g, p, x, wa, wb, wc, ba, bb, bc, y, ta, tb, ws, epi, fused_part, st);
    }
    if (s != QL_OK || !sp.on) return s;
    const int M = g.N * g.HO * g.WO;
    if (!sp.fused) {
        const dim3 grid(sp.nparts, cdiv(g.O, 64));
        if (g.dt == QL_BF16)
            hipLaunchKernelGGL(qconv_channel_stats_kernel<uint16_t>, grid, dim3(kThreads), 0, st,
                               static_cast<const uint16_t *>(y), M, g.O, sp.rpp, stat_part);
        else
            hipLaunchKernelGGL(qconv_channel_stats_kernel<float>, grid, dim3(kThreads), 0, st,
                               static_cast<const float *>(y), M, g.O, sp.rpp, stat_part);
        s = hip_status();
        if (s != QL_OK) return s;
    }
    hipLaunchKernelGGL(qconv_stats_reduce_kernel<>, dim3(2 * g.O), dim3(kThreads), 0, st, stat_part,
                       sp.nparts, g.O, e->sum, e->sumsq);
    return hip_status();
}

// x: the layer input X, used by the types whose terms see X o X (T2, where a
// NULL x falls back to X carried in `ta`, and T2&4, where it is required).
ql_status bwd_data_common(const Geom &g, const void *gy, const void *ta, const void *tb, const void *x,
                          const void *wa, const void *wb, const void *wc, void *dx, void *ws, size_t ws_bytes,
                          void *stream) {
    const int nt = g.terms();
    if (nt < 3) wc = nullptr;
    if (nt < 2) wb = nullptr;
    const void *xin = nullptr;
    if (g.ne == NEURON_T2) {
        xin = x ? x : ta;  // (T2 has no saved map: `ta` may carry X)
        ta = xin;
    } else if (g.ne == NEURON_T24) {
        xin = x;
        if (!xin) return QL_EINVAL;
    }
    if (g.om() == OM_SQUARE || g.om() == OM_SQIN) tb = nullptr;
    if (!gy || !ta || !wa || !dx || (nt >= 2 && (!tb || !wb)) || (nt >= 3 && !wc)) return QL_EINVAL;
    const void *ptrs[] = {gy, ta, tb, xin, wa, wb, wc, dx};
    for (const void *q : ptrs)
        if (q && !aligned16(q)) return QL_EINVAL;
    if (g.dw) {
        const void *w[3] = {wa, wb, wc};
        hipStream_t st = static_cast<hipStream_t>(stream);
        return run_dw_bwd_data(g, gy, ta, tb, w, dx, st);
    }
    const BwdDataPlan p = plan_bwd_data(g);
    if (ws_bytes < p.ws_bytes || (p.ws_bytes && !ws)) return QL_EWORKSPACE;
    if (ws && !aligned16(ws)) return QL_EINVAL;
    hipStream_t st = static_cast<hipStream_t>(stream);
    return run_bwd_data(g, p, gy, ta, tb, xin, wa, wb, wc, dx, ws, st);
}

// noalloc: the workspace is the library's scratch array (ws and ws_bytes are
// ignored); the split-K plan is capped to fit it.
ql_status bwd_weight_common(const Geom &g, const void *x, const void *gy, const void *ta, const void *tb,
                            float *dwa, float *dwb, float *dwc, float *dba, float *dbb, float *dbc, void *ws,
                            size_t ws_bytes, void *stream, bool noalloc = false) {
    const int nt = g.terms(), ngm = om_gmaps(g.om());
    // pointers of terms (and maps) the neuron type lacks are ignored
    if (nt < 3) { dwc = nullptr; dbc = nullptr; }
    if (nt < 2) { dwb = nullptr; dbb = nullptr; }
    if (ngm < 3) tb = nullptr;
    if (ngm < 2) ta = nullptr;
    if (!x || !gy || (ngm >= 2 && !ta) || (ngm >= 3 && !tb) || !dwa || (nt >= 2 && !dwb) || (nt >= 3 && !dwc))
        return QL_EINVAL;
    const int nb = (dba != nullptr) + (dbb != nullptr) + (dbc != nullptr);
    if (nb != 0 && nb != nt) return QL_EINVAL;
    const void *ptrs[] = {x, gy, ta, tb, dwa, dwb, dwc, dba, dbb, dbc};
    for (const void *q : ptrs)
        if (q && !aligned16(q)) return QL_EINVAL;
    if (g.dw) {
        const DwPlan p = plan_dw(g, 2);
        if (noalloc) {
            if (p.ws_bytes > kScratchBytes) return QL_EWORKSPACE;
            ws = scratch_ptr();
            ws_bytes = kScratchBytes;
            if (!ws) return QL_EHIP;
        }
        if (ws_bytes < p.ws_bytes || (p.ws_bytes && !ws)) return QL_EWORKSPACE;
        if (ws && !aligned16(ws)) return QL_EINVAL;
        float *const dw[3] = {dwa, dwb, dwc};
        float *const db[3] = {dba, dbb, dbc};
        hipStream_t st = static_cast<hipStream_t>(stream);
        return run_dw_bwd_weight(g, p, x, gy, ta, tb, dw, db, ws, st);
    }
    BwdWeightPlan p = plan_bwd_weight(g);
    if (noalloc) {
        // the regular plan where it fits (then the results are bitwise those of
        // the regular entry point), else fewer splits: dW and db partials of
        // 3 O (KP + 1) floats per split, two 256-byte alignments
        if (p.ws_bytes > kScratchBytes) {
            const size_t room = kScratchBytes - std::min(kScratchBytes, p.xpad_bytes + 2 * kAlign);
            const size_t kpo = (size_t)g.KH * g.KW * g.C;
            p = plan_bwd_weight(g, room / (kpo + 1) * kpo);
        }
        if (p.ws_bytes > kScratchBytes) return QL_EWORKSPACE;
        ws = scratch_ptr();
        ws_bytes = kScratchBytes;
        if (!ws) return QL_EHIP;
    }
    if (ws_bytes < p.ws_bytes || (p.ws_bytes && !ws)) return QL_EWORKSPACE;
    if (ws && !aligned16(ws)) return QL_EINVAL;
    hipStream_t st = static_cast<hipStream_t>(stream);
    return run_bwd_weight(g, p, x, gy, ta, tb, dwa, dwb, dwc, dba, dbb, dbc, ws, st);
}

// The layer's backward behind its ReLU (the fused epilogue's activation): G =
// gy o [y' > 0] into the front of the workspace, then the input gradient (dx
// non-NULL) and the weight and bias gradients (dwa non-NULL) from it, as the
// regular entry points compute them, in the rest.  Everything is validated
// before the first launch.
size_t bwd_relu_ws_bytes(const Geom &g, bool want_dx, bool want_dw) {
    const size_t gbytes = align_up((size_t)g.N * g.HO * g.WO * g.O * g.esize());
    size_t bd = 0, bw = 0;
    if (want_dx && !g.dw) bd = plan_bwd_data(g).ws_bytes;
    if (want_dw) bw = g.dw ? plan_dw(g, 2).ws_bytes : plan_bwd_weight(g).ws_bytes;
    return gbytes + std::max(bd, bw);
}

ql_status bwd_relu_common(const Geom &g, const void *x, const void *gy, const void *y_out, const void *ta,
                          const void *tb, const void *wa, const void *wb, const void *wc, void *dx, float *dwa,
                          float *dwb, float *dwc, float *dba, float *dbb, float *dbc, void *ws, size_t ws_bytes,
                          void *stream) {
    const int nt = g.terms(), ngm = om_gmaps(g.om());
    if (nt < 3) { wc = nullptr; dwc = nullptr; dbc = nullptr; }
    if (nt < 2) { wb = nullptr; dwb = nullptr; dbb = nullptr; }
    if (ngm < 3) tb = nullptr;
    if (ngm < 2) ta = nullptr;  // (T2's input gradient takes X itself)
    const int nw = (dwa != nullptr) + (dwb != nullptr) + (dwc != nullptr);
    const int nb = (dba != nullptr) + (dbb != nullptr) + (dbc != nullptr);
    if ((nw != 0 && nw != nt) || (nb != 0 && nb != nt) || (nb != 0 && nw == 0)) return QL_EINVAL;
    if (!dx && nw == 0) return QL_EINVAL;
    if (!x || !gy || !y_out || (ngm >= 2 && !ta) || (ngm >= 3 && !tb)) return QL_EINVAL;
    if (dx && (!wa || (nt >= 2 && !wb) || (nt >= 3 && !wc))) return QL_EINVAL;
    const void *ptrs[] = {x, gy, y_out, ta, tb, wa, wb, wc, dx, dwa, dwb, dwc, dba, dbb, dbc};
    for (const void *q : ptrs)
        if (q && !aligned16(q)) return QL_EINVAL;
    const size_t need = bwd_relu_ws_bytes(g, dx != nullptr, nw != 0);
    if (ws_bytes < need || !ws) return QL_EWORKSPACE;
    if (!aligned16(ws)) return QL_EINVAL;
    const size_t gbytes = align_up((size_t)g.N * g.HO * g.WO * g.O * g.esize());
    const long long n = (long long)g.N * g.HO * g.WO * g.O;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const int vec = g.vec();
    const int grid = grid_1d(std::max(1LL, n / vec));
    if (g.dt == QL_BF16)
        hipLaunchKernelGGL(qconv_relu_mask_kernel<uint16_t>, dim3(grid), dim3(kThreads), 0, st,
                           static_cast<const uint16_t *>(gy), static_cast<const uint16_t *>(y_out),
                           static_cast<uint16_t *>(ws), n);
    else
        hipLaunchKernelGGL(qconv_relu_mask_kernel<float>, dim3(grid), dim3(kThreads), 0, st,
                           static_cast<const float *>(gy), static_cast<const float *>(y_out),
                           static_cast<float *>(ws), n);
    ql_status s = hip_status();
    if (s != QL_OK) return s;
    const void *gm = ws;
    char *rest = static_cast<char *>(ws) + gbytes;
    const size_t rest_bytes = ws_bytes - gbytes;
    if (dx) {
        s = bwd_data_common(g, gm, g.ne == NEURON_T2 ? x : ta, tb, x, wa, wb, wc, dx, rest, rest_bytes, stream);
        if (s != QL_OK) return s;
    }
    if (nw) s = bwd_weight_common(g, x, gm, ta, tb, dwa, dwb, dwc, dba, dbb, dbc, rest, rest_bytes, stream);
    return s;
}

}  // namespace

extern "C" {

const char *qlayer_status_string(ql_status s) {
    switch (s) {
        case QL_OK: return "ok";
        case QL_EINVAL: return "invalid argument";
        case QL_EUNSUPPORTED: return "unsupported configuration";
        case QL_EWORKSPACE: return "workspace missing or too small";
        case QL_EHIP: return "HIP runtime error";
    }
    return "unknown status";
}

int qlayer_version(void) { return 100; }

size_t qlayer_conv2d_fwd_workspace_size(const ql_conv_desc *desc) {
    Geom g;
    if (make_geom(desc, g) != QL_OK) return 0;
    return fwd_ws_bytes(g, nullptr);
}

ql_status qlayer_conv2d_fwd(const ql_conv_desc *desc, const void *x, const void *wa, const void *wb, const void *wc,
                            const float *ba, const float *bb, const float *bc, void *y, void *ta, void *tb,
                            void *workspace, size_t workspace_bytes, void *stream) {
    Geom g;
    const ql_status s = make_geom(desc, g);
    if (s != QL_OK) return s;
    return fwd_common(g, x, wa, wb, wc, ba, bb, bc, y, ta, tb, nullptr, workspace, workspace_bytes, stream);
}

size_t qlayer_conv2d_bwd_data_workspace_size(const ql_conv_desc *desc) {
    Geom g;
    if (make_geom(desc, g) != QL_OK) return 0;
    if (g.dw) return 0;
    return plan_bwd_data(g).ws_bytes;
}

ql_status qlayer_conv2d_bwd_data(const ql_conv_desc *desc, const void *gy, const void *ta, const void *tb,
                                 const void *wa, const void *wb, const void *wc, void *dx, void *workspace,
                                 size_t workspace_bytes, void *stream) {
    Geom g;
    const ql_status s = make_geom(desc, g);
    if (s != QL_OK) return s;
    return bwd_data_common(g, gy, ta, tb, nullptr, wa, wb, wc, dx, workspace, workspace_bytes, stream);
}

ql_status qlayer_conv2d_bwd_data_ex(const ql_conv_desc *desc, const void *gy, const void *ta, const void *tb,
                                    const void *x, const void *wa, const void *wb, const void *wc, void *dx,
                                    void *workspace, size_t workspace_bytes, void *stream) {
    Geom g;
    const ql_status s = make_geom(desc, g);
    if (s != QL_OK) return s;
    return bwd_data_common(g, gy, ta, tb, x, wa, wb, wc, dx, workspace, workspace_bytes, stream);
}

size_t qlayer_conv2d_bwd_weight_workspace_size(const ql_conv_desc *desc) {
    Geom g;
    if (make_geom(desc, g) != QL_OK) return 0;
    if (g.dw) return plan_dw(g, 2).ws_bytes;
    return plan_bwd_weight(g).ws_bytes;
}

ql_status qlayer_conv2d_bwd_weight(const ql_conv_desc *desc, const void *x, const void *gy, const void *ta,
                                   const void *tb, float *dwa, float *dwb, float *dwc, float *dba, float *dbb,
                                   float *dbc, void *workspace, size_t workspace_bytes, void *stream) {
    Geom g;
    const ql_status s = make_geom(desc, g);
    if (s != QL_OK) return s;
    return bwd_weight_common(g, x, gy, ta, tb, dwa, dwb, dwc, dba, dbb, dbc, workspace, workspace_bytes, stream);
}

ql_status qlayer_conv2d_bwd_weight_noalloc(const ql_conv_desc *desc, const void *x, const void *gy, const void *ta,
                                           const void *tb, float *dwa, float *dwb, float *dwc, float *dba,
                                           float *dbb, float *dbc, void *stream) {
    Geom g;
    const ql_status s = make_geom(desc, g);
    if (s != QL_OK) return s;
    return bwd_weight_common(g, x, gy, ta, tb, dwa, dwb, dwc, dba, dbb, dbc, nullptr, 0, stream, true);
}

size_t qlayer_linear_fwd_workspace_size(const ql_linear_desc *desc) {
    Geom g;
    if (linear_geom(desc, g) != QL_OK) return 0;
    return fwd_ws_bytes(g, nullptr);
}

size_t qlayer_conv2d_fwd_ex_workspace_size(const ql_conv_desc *desc, const ql_epilogue *epi) {
    Geom g;
    if (make_geom(desc, g) != QL_OK) return 0;
    return fwd_ws_bytes(g, epi);
}

ql_status qlayer_conv2d_fwd_ex(const ql_conv_desc *desc, const void *x, const void *wa, const void *wb,
                               const void *wc, const float *ba, const float *bb, const float *bc, void *y, void *ta,
                               void *tb, const ql_epilogue *epi, void *workspace, size_t workspace_bytes,
                               void *stream) {
    Geom g;
    const ql_status s = make_geom(desc, g);
    if (s != QL_OK) return s;
    return fwd_common(g, x, wa, wb, wc, ba, bb, bc, y, ta, tb, epi, workspace, workspace_bytes, stream);
}

size_t qlayer_linear_fwd_ex_workspace_size(const ql_linear_desc *desc, const ql_epilogue *epi) {
    Geom g;
    if (linear_geom(desc, g) != QL_OK) return 0;
    return fwd_ws_bytes(g, epi);
}

ql_status qlayer_linear_fwd_ex(const ql_linear_desc *desc, const void *x, const void *wa, const void *wb,
                               const void *wc, const float *ba, const float *bb, const float *bc, void *y, void *ta,
                               void *tb, const ql_epilogue *epi, void *workspace, size_t workspace_bytes,
                               void *stream) {
    Geom g;
    const ql_status s = linear_geom(desc, g);
    if (s != QL_OK) return s;
    return fwd_common(g, x, wa, wb, wc, ba, bb, bc, y, ta, tb, epi, workspace, workspace_bytes, stream);
}

ql_status qlayer_linear_fwd(const ql_linear_desc *desc, const void *x, const void *wa, const void *wb,
                            const void *wc, const float *ba, const float *bb, const float *bc, void *y, void *ta,
                            void *tb, void *workspace, size_t workspace_bytes, void *stream) {
    Geom g;
    const ql_status s = linear_geom(desc, g);
    if (s != QL_OK) return s;
    return fwd_common(g, x, wa, wb, wc, ba, bb, bc, y, ta, tb, nullptr, workspace, workspace_bytes, stream);
}

size_t qlayer_linear_bwd_workspace_size(const ql_linear_desc *desc) {
    Geom g;
    if (linear_geom(desc, g) != QL_OK) return 0;
    return std::max(plan_bwd_data(g).ws_bytes, plan_bwd_weight(g).ws_bytes);
}

ql_status qlayer_linear_bwd(const ql_linear_desc *desc, const void *x, const void *gy, const void *ta,
                            const void *tb, const void *wa, const void *wb, const void *wc, void *dx, float *dwa,
                            float *dwb, float *dwc, float *dba, float *dbb, float *dbc, void *workspace,
                            size_t workspace_bytes, void *stream) {
    Geom g;
    ql_status s = linear_geom(desc, g);
    if (s != QL_OK) return s;
    const int nt = g.terms(), ngm = om_gmaps(g.om());
    // pointers of terms (and maps) the neuron type lacks are ignored
    if (nt < 3) { wc = nullptr; dwc = nullptr; dbc = nullptr; }
    if (nt < 2) { wb = nullptr; dwb = nullptr; dbb = nullptr; }
    if (ngm < 3) tb = nullptr;
    if (ngm < 2) ta = nullptr;
    const int nw = (dwa != nullptr) + (dwb != nullptr) + (dwc != nullptr);
    const int nb = (dba != nullptr) + (dbb != nullptr) + (dbc != nullptr);
    if ((nw != 0 && nw != nt) || (nb != 0 && nb != nt) || (nb != 0 && nw == 0)) return QL_EINVAL;
    if (!dx && nw == 0) return QL_EINVAL;
    if (!x || !gy || (ngm >= 2 && !ta) || (ngm >= 3 && !tb) || !wa || (nt >= 2 && !wb) || (nt >= 3 && !wc))
        return QL_EINVAL;
    // Validate everything before the first launch.
    const void *ptrs[] = {x, gy, ta, tb, wa, wb, wc, dx, dwa, dwb, dwc, dba, dbb, dbc};
    for (const void *q : ptrs)
        if (q && !aligned16(q)) return QL_EINVAL;
    const size_t need = std::max(dx ? plan_bwd_data(g).ws_bytes : 0, nw ? plan_bwd_weight(g).ws_bytes : 0);
    if (workspace_bytes < need || (need && !workspace)) return QL_EWORKSPACE;
    if (dx) {
        // (T2: the input gradient takes X in place of the saved map)
        s = bwd_data_common(g, gy, ta, tb, x, wa, wb, wc, dx, workspace, workspace_bytes, stream);
        if (s != QL_OK) return s;
    }
    if (nw) s = bwd_weight_common(g, x, gy, ta, tb, dwa, dwb, dwc, dba, dbb, dbc, workspace, workspace_bytes, stream);
    return s;
}

size_t qlayer_conv2d_bwd_relu_workspace_size(const ql_conv_desc *desc) {
    Geom g;
    if (make_geom(desc, g) != QL_OK) return 0;
    return bwd_relu_ws_bytes(g, true, true);
}

ql_status qlayer_conv2d_bwd_relu(const ql_conv_desc *desc, const void *x, const void *gy, const void *y_out,
                                 const void *ta, const void *tb, const void *wa, const void *wb, const void *wc,
                                 void *dx, float *dwa, float *dwb, float *dwc, float *dba, float *dbb, float *dbc,
                                 void *workspace, size_t workspace_bytes, void *stream) {
    Geom g;
    const ql_status s = make_geom(desc, g);
    if (s != QL_OK) return s;
    return bwd_relu_common(g, x, gy, y_out, ta, tb, wa, wb, wc, dx, dwa, dwb, dwc, dba, dbb, dbc, workspace,
                           workspace_bytes, stream);
}

size_t qlayer_linear_bwd_relu_workspace_size(const ql_linear_desc *desc) {
    Geom g;
    if (linear_geom(desc, g) != QL_OK) return 0;
    return bwd_relu_ws_bytes(g, true, true);
}

ql_status qlayer_linear_bwd_relu(const ql_linear_desc *desc, const void *x, const void *gy, const void *y_out,
                                 const void *ta, const void *tb, const void *wa, const void *wb, const void *wc,
                                 void *dx, float *dwa, float *dwb, float *dwc, float *dba, float *dbb, float *dbc,
                                 void *workspace, size_t workspace_bytes, void *stream) {
    Geom g;
    const ql_status s = linear_geom(desc, g);
    if (s != QL_OK) return s;
    return bwd_relu_common(g, x, gy, y_out, ta, tb, wa, wb, wc, dx, dwa, dwb, dwc, dba, dbb, dbc, workspace,
                           workspace_bytes, stream);
}

}  // extern "C"
