/*
 * qnet.h -- C ABI of the network glue around the quadratic layers, for the
 * CIFAR ResNet training step (arXiv 2204.01701, section 4.2, model
 * construction: batch normalization after the quadratic layers, a ReLU in
 * deeper networks; residual blocks; the classifier after global average
 * pooling).  Exported by libqlayer.so beside the layer entry points of
 * qlayer.h, with the same conventions: device pointers owned by the caller,
 * 16-byte aligned; NHWC tensors of `dtype` (float32, or bfloat16 stored as
 * uint16) with fp32 arithmetic; per-channel statistics float32; work enqueued
 * on `stream`; arguments validated on the host before any launch (QL_EINVAL),
 * QL_EHIP on a launch error.  Channel counts must be multiples of 4.
 *
 * Batch normalization is in training mode with gamma = 1 and beta = 0, its
 * batch statistics taken from the per-channel sums S = sum y, Q = sum y^2
 * over the M = N H W pixels that qlayer_conv2d_fwd_ex gathers from the
 * stored y:  mean = S / M,  var = Q / M - mean^2,  rstd = 1 / sqrt(var + eps).
 */
#ifndef QNET_H
#define QNET_H

#include <stddef.h>

#include "qlayer.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct { int n, h, w, c; } qnet_shape; /* an NHWC tensor */

/* Forward of batch normalization, the optional shortcut and the optional ReLU:
 *   out = relu((y - mean) rstd + r)       (relu != 0; else without the clamp)
 *   s      : shape of y and out.
 *   sum, sumsq : the per-channel sums of y (C floats each).
 *   res    : the shortcut r, or NULL (none): rs == s (identity), or the
 *            option-A shortcut of a stride-2 transition: rs = (n, 2h, 2w, c / 2),
 *            the input subsampled by 2 and placed at channels [c/4, c/4 + c/2),
 *            zeros elsewhere.  Other shapes: QL_EINVAL.
 *   mean, rstd : written (C floats each), for the backward. */
ql_status qnet_bn_act_fwd(const qnet_shape *s, ql_dtype dtype, const void *y, const float *sum,
                          const float *sumsq, float eps, const void *res, const qnet_shape *rs, int relu,
                          void *out, float *mean, float *rstd, void *stream);

/* Backward of qnet_bn_act_fwd up to y: with dz = dout [out > 0] (relu != 0;
 * else dz = dout) and x^ = (y - mean) rstd,
 *   dy = rstd (dz - sum(dz) / M - x^ sum(dz x^) / M)
 * (the shortcut's gradient is added by qnet_residual_bwd).  The per-channel
 * sums are reduced in a fixed order (deterministic).  workspace: at least
 * qnet_bn_act_bwd_workspace_size(s) bytes. */
size_t qnet_bn_act_bwd_workspace_size(const qnet_shape *s);
ql_status qnet_bn_act_bwd(const qnet_shape *s, ql_dtype dtype, const void *dout, const void *out, int relu,
                          const void *y, const float *mean, const float *rstd, void *dy, void *workspace,
                          size_t workspace_bytes, void *stream);

/* The shortcut's gradient added to the block input's: dx (shape xs, the input
 * gradient of the block's first layer) += the shortcut's share of
 * dz = dout [out > 0] (shape s, the block output): dz itself when xs == s,
 * the option-A gather when xs = (n, 2h, 2w, c / 2). */
ql_status qnet_residual_bwd(const qnet_shape *s, ql_dtype dtype, const void *dout, const void *out,
                            const qnet_shape *xs, void *dx, void *stream);

/* Global average pooling of x (shape s) to y (s.n x s.c), and its backward. */
ql_status qnet_gap_fwd(const qnet_shape *s, ql_dtype dtype, const void *x, void *y, void *stream);
ql_status qnet_gap_bwd(const qnet_shape *s, ql_dtype dtype, const void *dy, void *dx, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* QNET_H */
