// qnet.hip -- host side of the network glue ABI (include/qnet.h): argument
// checks and the launches of the kernels in qnet_glue.h.
#include "qnet.h"
#include "qhost.h"
#include "qnet_glue.h"

using namespace ql;
using namespace ql::host;

namespace {

bool shape_ok(const qnet_shape *s) {
    return s && s->n > 0 && s->h > 0 && s->w > 0 && s->c > 0 && s->c % 4 == 0 &&
           (long long)s->n * s->h * s->w * s->c <= (1LL << 31) - 1;
}
bool dtype_ok(ql_dtype d) { return d == QL_F32 || d == QL_BF16; }
NetShape ns(const qnet_shape *s) { return NetShape{s->n, s->h, s->w, s->c}; }
long long pixels(const qnet_shape *s) { return (long long)s->n * s->h * s->w; }

int grid_for(long long items) {
    const long long b = (items + kThreads - 1) / kThreads;
    return (int)std::max(1LL, std::min(b, 16LL * kNumCUs));
}

// rows per part of the backward reduction (at least 64, at most 1024 parts)
int bwd_rpp(const qnet_shape *s) { return std::max(64, cdiv(pixels(s), 1024)); }
int bwd_parts(const qnet_shape *s) { return cdiv(pixels(s), bwd_rpp(s)); }

}  // namespace

extern "C" {

ql_status qnet_bn_act_fwd(const qnet_shape *s, ql_dtype dtype, const void *y, const float *sum, const float *sumsq,
                          float eps, const void *res, const qnet_shape *rs, int relu, void *out, float *mean,
                          float *rstd, void *stream) {
    if (!shape_ok(s) || !dtype_ok(dtype) || !(eps >= 0.0f)) return QL_EINVAL;
    if (!y || !sum || !sumsq || !out || !mean || !rstd) return QL_EINVAL;
    int mode = RES_NONE;
    NetShape r{0, 0, 0, 0};
    if (res) {
        if (!rs || rs->n != s->n) return QL_EINVAL;
        if (rs->h == s->h && rs->w == s->w && rs->c == s->c) mode = RES_SAME;
        else if (rs->h == 2 * s->h && rs->w == 2 * s->w && 2 * rs->c == s->c && s->c % 16 == 0) mode = RES_SUB2;
        else return QL_EINVAL;
        r = ns(rs);
    }
    const void *ptrs[] = {y, sum, sumsq, res, out, mean, rstd};
    for (const void *q : ptrs)
        if (q && !aligned16(q)) return QL_EINVAL;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const dim3 grid(grid_for(pixels(s) * s->c / 4));
    if (dtype == QL_BF16)
        hipLaunchKernelGGL(qnet_bn_act_fwd_kernel<uint16_t>, grid, dim3(kThreads), 0, st, ns(s),
                           static_cast<const uint16_t *>(y), sum, sumsq, eps, mode,
                           static_cast<const uint16_t *>(res), r, relu, static_cast<uint16_t *>(out), mean, rstd);
    else
        hipLaunchKernelGGL(qnet_bn_act_fwd_kernel<float>, grid, dim3(kThreads), 0, st, ns(s),
                           static_cast<const float *>(y), sum, sumsq, eps, mode, static_cast<const float *>(res), r,
                           relu, static_cast<float *>(out), mean, rstd);
    return hip_status();
}

size_t qnet_bn_act_bwd_workspace_size(const qnet_shape *s) {
    if (!shape_ok(s)) return 0;
    // per-part partial sums [part][2][C], then the two reduced sums [2][C]
    return align_up((size_t)bwd_parts(s) * 2 * s->c * sizeof(float)) + align_up((size_t)2 * s->c * sizeof(float));
}

ql_status qnet_bn_act_bwd(const qnet_shape *s, ql_dtype dtype, const void *dout, const void *out, int relu,
                          const void *y, const float *mean, const float *rstd, void *dy, void *workspace,
                          size_t workspace_bytes, void *stream) {
    if (!shape_ok(s) || !dtype_ok(dtype)) return QL_EINVAL;
    if (!dout || !out || !y || !mean || !rstd || !dy) return QL_EINVAL;
    const void *ptrs[] = {dout, out, y, mean, rstd, dy, workspace};
    for (const void *q : ptrs)
        if (q && !aligned16(q)) return QL_EINVAL;
    const size_t need = qnet_bn_act_bwd_workspace_size(s);
    if (!workspace || workspace_bytes < need) return QL_EWORKSPACE;
    const int rpp = bwd_rpp(s), parts = bwd_parts(s);
    float *part = static_cast<float *>(workspace);
    float *sums = reinterpret_cast<float *>(static_cast<char *>(workspace) +
                                            align_up((size_t)parts * 2 * s->c * sizeof(float)));
    hipStream_t st = static_cast<hipStream_t>(stream);
    const dim3 rgrid(parts, cdiv(s->c, 64));
    const dim3 agrid(grid_for(pixels(s) * s->c / 4));
    if (dtype == QL_BF16) {
        using T = uint16_t;
        hipLaunchKernelGGL(qnet_bn_act_bwd_reduce_kernel<T>, rgrid, dim3(kThreads), 0, st, ns(s),
                           static_cast<const T *>(dout), static_cast<const T *>(out), relu, static_cast<const T *>(y),
                           mean, rstd, rpp, part);
        hipLaunchKernelGGL(qconv_stats_reduce_kernel<>, dim3(2 * s->c), dim3(kThreads), 0, st, part, parts,
                           s->c, sums, sums + s->c);
        hipLaunchKernelGGL(qnet_bn_act_bwd_apply_kernel<T>, agrid, dim3(kThreads), 0, st, ns(s),
                           static_cast<const T *>(dout), static_cast<const T *>(out), relu, static_cast<const T *>(y),
                           mean, rstd, sums, sums + s->c, static_cast<T *>(dy));
    } else {
        using T = float;
        hipLaunchKernelGGL(qnet_bn_act_bwd_reduce_kernel<T>, rgrid, dim3(kThreads), 0, st, ns(s),
                           static_cast<const T *>(dout), static_cast<const T *>(out), relu, static_cast<const T *>(y),
                           mean, rstd, rpp, part);
        hipLaunchKernelGGL(qconv_stats_reduce_kernel<>, dim3(2 * s->c), dim3(kThreads), 0, st, part, parts,
                           s->c, sums, sums + s->c);
        hipLaunchKernelGGL(qnet_bn_act_bwd_apply_kernel<T>, agrid, dim3(kThreads), 0, st, ns(s),
                           static_cast<const T *>(dout), static_cast<const T *>(out), relu, static_cast<const T *>(y),
                           mean, rstd, sums, sums + s->c, static_cast<T *>(dy));
    }
    return hip_status();
}

ql_status qnet_residual_bwd(const qnet_shape *s, ql_dtype dtype, const void *dout, const void *out,
                            const qnet_shape *xs, void *dx, void *stream) {
    if (!shape_ok(s) || !shape_ok(xs) || !dtype_ok(dtype) || !dout || !out || !dx || xs->n != s->n)
        return QL_EINVAL;
    int mode;
    if (xs->h == s->h && xs->w == s->w && xs->c == s->c) mode = RES_SAME;
    else if (xs->h == 2 * s->h && xs->w == 2 * s->w && 2 * xs->c == s->c && s->c % 16 == 0) mode = RES_SUB2;
    else return QL_EINVAL;
    const void *ptrs[] = {dout, out, dx};
    for (const void *q : ptrs)
        if (!aligned16(q)) return QL_EINVAL;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const dim3 grid(grid_for(pixels(xs) * xs->c / 4));
    if (dtype == QL_BF16)
        hipLaunchKernelGGL(qnet_residual_bwd_kernel<uint16_t>, grid, dim3(kThreads), 0, st, ns(s),
                           static_cast<const uint16_t *>(dout), static_cast<const uint16_t *>(out), ns(xs), mode,
                           static_cast<uint16_t *>(dx));
    else
        hipLaunchKernelGGL(qnet_residual_bwd_kernel<float>, grid, dim3(kThreads), 0, st, ns(s),
                           static_cast<const float *>(dout), static_cast<const float *>(out), ns(xs), mode,
                           static_cast<float *>(dx));
    return hip_status();
}

ql_status qnet_gap_fwd(const qnet_shape *s, ql_dtype dtype, const void *x, void *y, void *stream) {
    if (!shape_ok(s) || !dtype_ok(dtype) || !x || !y || !aligned16(x) || !aligned16(y)) return QL_EINVAL;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const dim3 grid(cdiv((long long)s->n * s->c, kThreads));
    if (dtype == QL_BF16)
        hipLaunchKernelGGL(qnet_gap_fwd_kernel<uint16_t>, grid, dim3(kThreads), 0, st, ns(s),
                           static_cast<const uint16_t *>(x), static_cast<uint16_t *>(y));
    else
        hipLaunchKernelGGL(qnet_gap_fwd_kernel<float>, grid, dim3(kThreads), 0, st, ns(s),
                           static_cast<const float *>(x), static_cast<float *>(y));
    return hip_status();
}

ql_status qnet_gap_bwd(const qnet_shape *s, ql_dtype dtype, const void *dy, void *dx, void *stream) {
    if (!shape_ok(s) || !dtype_ok(dtype) || !dy || !dx || !aligned16(dy) || !aligned16(dx)) return QL_EINVAL;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const dim3 grid(grid_for(pixels(s) * s->c));
    if (dtype == QL_BF16)
        hipLaunchKernelGGL(qnet_gap_bwd_kernel<uint16_t>, grid, dim3(kThreads), 0, st, ns(s),
                           static_cast<const uint16_t *>(dy), static_cast<uint16_t *>(dx));
    else
        hipLaunchKernelGGL(qnet_gap_bwd_kernel<float>, grid, dim3(kThreads), 0, st, ns(s),
                           static_cast<const float *>(dy), static_cast<float *>(dx));
    return hip_status();
}

}  // extern "C"
