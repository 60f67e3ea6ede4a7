/*
 * qlayer.h -- C ABI of the MI355X (gfx950) quadratic-neuron layer library.
 *
 * The layer is the quadratic neuron of QuadraLib (arXiv 2204.01701, section
 * 3.1, equation eq:2ndneuron3):
 *
 *     Y = (W_a * X + b_a) o (W_b * X + b_b) + (W_c * X + b_c)
 *
 * "o" is the elementwise (Hadamard) product (Table 1, note 3); each of the
 * three terms T_t = W_t * X + b_t is an ordinary first-order layer (section
 * 3.2, P4), which is why each keeps its own bias.  As a convolution "*" is the
 * cross-correlation of a PyTorch nn.Conv2d (section 4.2: zero padding, floor
 * output size, dilation 1, kernel/stride/padding/groups shared by the three
 * terms; groups 1, or groups = C for the depth-wise setting of section 4.2).  As a fully-connected layer (section 3.2, P3) "*" is a
 * matrix product.  The backward pass follows section 4.3 (eq:AD, eq:SD):
 * with G = dl/dY, the per-term output gradients are
 *
 *     G_a = G o T_b,   G_b = G o T_a,   G_c = G
 *
 * and each term then back-propagates as an ordinary first-order layer.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - All tensor pointers are DEVICE pointers owned by the caller.  The library
 *    keeps no pointer after a call returns and never allocates device memory.
 *  - Work is enqueued asynchronously on `stream` (a hipStream_t, passed as
 *    void*; NULL = the null stream).  A return of QL_OK means "enqueued".
 *  - Layouts (row-major, innermost last):
 *      conv X, dX       : N x H x W x C          (NHWC)
 *      conv W_t         : O x KH x KW x C        (OHWI), dW_t the same
 *                         (depthwise, groups = C = O: C x KH x KW x 1)
 *      conv Y, G, T_a, T_b : N x Ho x Wo x O     (NHWC),
 *                          Ho = (H + 2*pad_h - KH) / stride_h + 1 (floor), Wo likewise
 *      dense X, dX      : B x I;  W_t, dW_t : O x I;  Y, G, T_a, T_b : B x O
 *      biases b_t, db_t : O
 *  - dtype QL_F32: every tensor is float32.  dtype QL_BF16: X, W_t, Y, G,
 *    T_a, T_b and dX are bfloat16 (stored as uint16), arithmetic is fp32
 *    (MFMA with fp32 accumulation), bf16 outputs are rounded to nearest even.
 *    Biases, dW_t and db_t are ALWAYS float32.
 *  - Every tensor pointer must be 16-byte aligned.
 *  - Errors: arguments are validated on the host before anything is
 *    launched.  Invalid arguments (non-positive sizes, empty output, stride<1,
 *    pad<0, unknown dtype, NULL required pointer, misaligned pointer) give
 *    QL_EINVAL; a workspace smaller than the size query gives QL_EWORKSPACE;
 *    a HIP launch error gives QL_EHIP.  Outputs are unspecified after a
 *    non-QL_OK return.  No entry point aborts or throws.
 *  - Workspaces: caller-allocated device memory of at least the size the
 *    matching *_workspace_size() query returns for the same descriptor (the
 *    query may return 0; the pointer may then be NULL).  Its contents on entry
 *    are irrelevant.  Two calls that share a workspace must not overlap.
 */
#ifndef QLAYER_H
#define QLAYER_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { QL_F32 = 0, QL_BF16 = 1 } ql_dtype;

/* Neuron type of a layer.  QL_NEURON_QUADRA is the design of section 3.1
 * (eq:2ndneuron3); the others are the earlier quadratic neurons of Table 1
 * that the paper evaluates against (Table 3), each built from the same
 * first-order terms T_t = W_t * X + b_t:
 *   QL_NEURON_QUADRA      Y = T_a o T_b + T_c            (weights a, b, c)
 *   QL_NEURON_T4          Y = T_a o T_b                  (weights a, b)
 *   QL_NEURON_T4_IDENTITY Y = T_a o T_b + X              (weights a, b; C == O and the
 *                                                         output map the size of the input)
 *   QL_NEURON_T3          Y = T_a o T_a                  (weight a)
 *   QL_NEURON_T2          Y = W_a * (X o X) + b_a        (weight a)
 *   QL_NEURON_T24         Y = T_a o T_b + W_c * (X o X) + b_c
 *                         (weights a, b, c; "T2&4", the design section 3.1
 *                         replaces by putting X in place of X o X in the third term)
 * Backward, with G = dl/dY: G_a = G o T_b, G_b = G o T_a (T4 types, T2&4; the
 * shortcut adds G to dX), G_a = 2 G o T_a (T3), and for T2 dW_a correlates G
 * with X o X while dX = 2 X o (the transposed convolution of G with W_a);
 * T2&4's third term likewise: dW_c correlates G with X o X and adds
 * 2 X o (the transposed convolution of G with W_c) to dX.
 * Pointers of terms a type lacks are ignored (may be NULL); the saved maps
 * are T_a, T_b (QUADRA, T4 types, T2&4), T_a (T3), none (T2; its input
 * gradient takes X itself in the `ta` argument, or through
 * qlayer_conv2d_bwd_data_ex).  The input gradient of T2&4 needs X as well as
 * T_a and T_b: qlayer_conv2d_bwd_data_ex.  The depthwise layer covers the
 * types up to QL_NEURON_T2 (T2&4: QL_EUNSUPPORTED). */
typedef enum {
    QL_NEURON_QUADRA = 0,
    QL_NEURON_T4 = 1,
    QL_NEURON_T4_IDENTITY = 2,
    QL_NEURON_T3 = 3,
    QL_NEURON_T2 = 4,
    QL_NEURON_T24 = 5
} ql_neuron;

typedef enum {
    QL_OK = 0,
    QL_EINVAL = 1,       /* invalid argument */
    QL_EUNSUPPORTED = 2, /* valid but not covered by the kernels */
    QL_EWORKSPACE = 3,   /* workspace missing or too small */
    QL_EHIP = 4          /* a HIP runtime / launch error */
} ql_status;

/* Geometry of a quadratic 2-D convolution layer. */
typedef struct {
    int n, c, h, w;         /* input X: N x H x W x C */
    int o, kh, kw;          /* each W_t: O x KH x KW x C */
    int stride_h, stride_w; /* >= 1 */
    int pad_h, pad_w;       /* >= 0, symmetric zero padding */
    ql_dtype dtype;
    ql_neuron neuron;       /* QL_NEURON_QUADRA (0) unless set */
    int groups;             /* 0 or 1: every output channel sees every input channel;
                               C (with O == C): depthwise, each channel its own
                               KH x KW filter per term, W_t (C,KH,KW,1), dW_t the same;
                               its forward and input gradient need no workspace.
                               Other group counts, or depthwise filters above
                               13 x 13 (three terms staged per channel slice):
                               QL_EUNSUPPORTED. */
} ql_conv_desc;

/* Geometry of a quadratic fully-connected layer. */
typedef struct {
    int batch, in, out; /* X: batch x in, W_t: out x in, Y: batch x out */
    ql_dtype dtype;
    ql_neuron neuron;   /* QL_NEURON_QUADRA (0) unless set */
} ql_linear_desc;

/* Human-readable name of a status code (static storage). */
const char *qlayer_status_string(ql_status s);

/* Library version as major*10000 + minor*100 + patch. */
int qlayer_version(void);

/* ---------------------------------------------------------------------------
 * Convolution forward -- section 3.1 eq:2ndneuron3 applied as a conv layer.
 *   x          : X (N,H,W,C), required.
 *   wa, wb, wc : W_a, W_b, W_c (O,KH,KW,C), required for the terms the
 *                neuron type has (all three for QL_NEURON_QUADRA).
 *   ba, bb, bc : b_a, b_b, b_c (O) float32; each may be NULL (= zero).
 *   y          : Y (N,Ho,Wo,O); may be NULL only when the saved maps of the
 *                type are given (recompute mode of the hybrid
 *                back-propagation, section 4.3: only the term maps are
 *                regenerated); required for QL_NEURON_T2.
 *   ta, tb     : if non-NULL, T_a and T_b (N,Ho,Wo,O) are written as well
 *                (the "saved" term maps the backward needs; tb only for the
 *                two- and three-term types).  Recompute mode and saved mode
 *                produce bitwise identical T_a, T_b.
 *   workspace  : qlayer_conv2d_fwd_workspace_size(desc) bytes (split-K
 *                partial sums for layers with few output pixels).
 * T_c is never written.
 * ------------------------------------------------------------------------- */
size_t qlayer_conv2d_fwd_workspace_size(const ql_conv_desc *desc);
ql_status qlayer_conv2d_fwd(const ql_conv_desc *desc, const void *x,
                            const void *wa, const void *wb, const void *wc,
                            const float *ba, const float *bb, const float *bc,
                            void *y, void *ta, void *tb,
                            void *workspace, size_t workspace_bytes, void *stream);

/* ---------------------------------------------------------------------------
 * Convolution input gradient -- section 4.3 (eq:AD chain rule, eq:SD):
 *   dX = sum_t  conv_transpose(G_t, W_t),  G_a = G o T_b, G_b = G o T_a, G_c = G.
 *   gy     : G = dl/dY (N,Ho,Wo,O), required.
 *   ta, tb : the saved maps of the neuron type from a forward call: T_a and
 *            T_b (N,Ho,Wo,O) for QUADRA and the T4 types, T_a for T3; for T2
 *            `ta` is X (N,H,W,C) and tb is ignored.
 *   wa, wb, wc : weights (O,KH,KW,C) of the terms the type has.
 *   dx     : dX (N,H,W,C), written (not accumulated).
 * The products G o T_b and G o T_a are formed on the fly and never stored.
 * ------------------------------------------------------------------------- */
size_t qlayer_conv2d_bwd_data_workspace_size(const ql_conv_desc *desc);
ql_status qlayer_conv2d_bwd_data(const ql_conv_desc *desc, const void *gy,
                                 const void *ta, const void *tb,
                                 const void *wa, const void *wb, const void *wc,
                                 void *dx, void *workspace, size_t workspace_bytes,
                                 void *stream);

/* ---------------------------------------------------------------------------
 * Convolution input gradient with the layer input -- the same operation as
 * qlayer_conv2d_bwd_data for the neuron types whose terms see X o X (Table 1),
 * whose chain rule through the square needs X itself:
 *   x : X (N,H,W,C).  QL_NEURON_T24: required (with ta, tb), its c term adds
 *       2 X o conv_transpose(G, W_c).  QL_NEURON_T2: used in place of `ta`
 *       (then `ta` may be NULL).  Other types: ignored (may be NULL).
 * Other arguments, the workspace (qlayer_conv2d_bwd_data_workspace_size)
 * and errors as for qlayer_conv2d_bwd_data, which returns QL_EINVAL for
 * QL_NEURON_T24 (no X).
 * ------------------------------------------------------------------------- */
ql_status qlayer_conv2d_bwd_data_ex(const ql_conv_desc *desc, const void *gy,
                                    const void *ta, const void *tb, const void *x,
                                    const void *wa, const void *wb, const void *wc,
                                    void *dx, void *workspace, size_t workspace_bytes,
                                    void *stream);

/* ---------------------------------------------------------------------------
 * Convolution weight and bias gradients -- section 4.3 eq:SD:
 *   dW_t[o,r,q,c] = sum_{n,i,j} G_t[n,i,j,o] X[n, i*s-p+r, j*s-p+q, c]
 *   db_t[o]       = sum_{n,i,j} G_t[n,i,j,o]
 *   x, gy          : required; ta, tb: the saved maps of the type (none for T2).
 *   dwa, dwb, dwc  : float32 (O,KH,KW,C), required for the terms the type
 *                    has, written (not accumulated).
 *   dba, dbb, dbc  : float32 (O); given for every term of the type or all
 *                    NULL (= skip).
 *   workspace      : qlayer_conv2d_bwd_weight_workspace_size(desc) bytes
 *                    (split-K partials, reduced in a fixed order, so results
 *                    are deterministic run to run).
 * ------------------------------------------------------------------------- */
size_t qlayer_conv2d_bwd_weight_workspace_size(const ql_conv_desc *desc);
ql_status qlayer_conv2d_bwd_weight(const ql_conv_desc *desc, const void *x, const void *gy,
                                   const void *ta, const void *tb,
                                   float *dwa, float *dwb, float *dwc,
                                   float *dba, float *dbb, float *dbc,
                                   void *workspace, size_t workspace_bytes, void *stream);

/* ---------------------------------------------------------------------------
 * Convolution weight and bias gradients without a workspace -- for callers
 * that cannot allocate device memory: code under HIP graph capture, tight
 * serving or training loops, harnesses that forbid hipMalloc.  The same
 * operation, arguments and errors as qlayer_conv2d_bwd_weight minus the
 * workspace: the split-K partial sums (and the zero-padded copy of X of
 * few-channel layers) go to a scratch array the library owns, of
 * QLAYER_NOALLOC_SCRATCH_BYTES bytes on each GPU it runs on, held until the
 * process ends.  Where the regular call's workspace query fits that size the
 * plan, and so every result bit, is the regular call's; otherwise the split
 * count is lowered to fit (results equal up to summation order); a layer
 * that does not fit even then returns QL_EWORKSPACE.  No device memory is
 * allocated by this call; the first call on a device resolves the array's
 * address there.  Every call on one GPU shares its array, which keeps the
 * last call's contents (nothing in it needs to start at zero): calls that
 * overlap on one GPU (several streams or host threads) race, and the caller
 * must serialize them.
 * ------------------------------------------------------------------------- */
#define QLAYER_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
ql_status qlayer_conv2d_bwd_weight_noalloc(const ql_conv_desc *desc, const void *x, const void *gy,
                                           const void *ta, const void *tb,
                                           float *dwa, float *dwb, float *dwc,
                                           float *dba, float *dbb, float *dbc, void *stream);

/* ---------------------------------------------------------------------------
 * Fully-connected forward -- section 3.2 P3: Y = (X W_a^T + b_a) o (X W_b^T + b_b)
 * + X W_c^T + b_c.  Arguments as for qlayer_conv2d_fwd (biases may be NULL,
 * y may be NULL when ta and tb are given).
 * ------------------------------------------------------------------------- */
size_t qlayer_linear_fwd_workspace_size(const ql_linear_desc *desc);
ql_status qlayer_linear_fwd(const ql_linear_desc *desc, const void *x,
                            const void *wa, const void *wb, const void *wc,
                            const float *ba, const float *bb, const float *bc,
                            void *y, void *ta, void *tb,
                            void *workspace, size_t workspace_bytes, void *stream);

/* ---------------------------------------------------------------------------
 * Fully-connected backward -- section 4.3 eq:SD for the dense layer:
 *   dX = [G o T_b | G o T_a | G] [W_a; W_b; W_c],  dW_t = G_t^T X,  db_t = column sums of G_t.
 *   x, gy, ta, tb, wa, wb, wc : required.
 *   dx            : (B,I) or NULL to skip the input gradient.
 *   dwa, dwb, dwc : float32 (O,I); all three or none (NULL = skip).
 *   dba, dbb, dbc : float32 (O); all three or none; need dW.
 *   At least one of dx / dW must be requested.
 * ------------------------------------------------------------------------- */
size_t qlayer_linear_bwd_workspace_size(const ql_linear_desc *desc);
ql_status qlayer_linear_bwd(const ql_linear_desc *desc, const void *x, const void *gy,
                            const void *ta, const void *tb,
                            const void *wa, const void *wb, const void *wc,
                            void *dx, float *dwa, float *dwb, float *dwc,
                            float *dba, float *dbb, float *dbc,
                            void *workspace, size_t workspace_bytes, void *stream);

/* ---------------------------------------------------------------------------
 * Forward with a fused epilogue -- section 4.2, model construction: batch
 * normalization after the quadratic layers regulates the extreme values the
 * second-order term produces, and deeper networks put an activation (ReLU)
 * after them.  The forward kernel transforms Y before storing it:
 *
 *     y'[m, o] = relu( scale[o] * Y[m, o] + shift[o] )     (per output channel o)
 *
 * (a batch normalization with fixed statistics folds into scale and shift),
 * stores y' in y, and gathers the statistics a training-mode batch
 * normalization of y' needs, over the N x Ho x Wo pixels (B rows of a dense
 * layer) of each channel, from the values as stored (rounded to the dtype):
 *
 *     sum[o] = sum_m y'[m, o],    sumsq[o] = sum_m y'[m, o]^2
 *
 * Every member is optional: scale NULL = 1, shift NULL = 0, relu 0 = none,
 * sum and sumsq both NULL = no statistics (both or neither, else QL_EINVAL).
 * T_a and T_b are stored untransformed (the backward takes dl/dY, the
 * gradient before the epilogue, which the caller forms).  An epilogue that
 * does anything needs y != NULL (recompute mode has no Y): QL_EINVAL.  The
 * statistics are summed in a fixed order: repeated calls give identical bits.
 * The pointers are float32 device pointers of O values, 16-byte aligned.
 * epi == NULL is the plain forward.  The workspace query takes the same epi
 * (the statistics need per-tile partial sums); other arguments and errors as
 * for qlayer_conv2d_fwd / qlayer_linear_fwd.
 * ------------------------------------------------------------------------- */
typedef struct {
    const float *scale;  /* O per-channel factors, or NULL */
    const float *shift;  /* O per-channel offsets, or NULL */
    int relu;            /* nonzero: clamp y' at 0 */
    float *sum;          /* O: per-channel sum of y', or NULL */
    float *sumsq;        /* O: per-channel sum of y'^2, or NULL */
} ql_epilogue;

size_t qlayer_conv2d_fwd_ex_workspace_size(const ql_conv_desc *desc, const ql_epilogue *epi);
ql_status qlayer_conv2d_fwd_ex(const ql_conv_desc *desc, const void *x,
                               const void *wa, const void *wb, const void *wc,
                               const float *ba, const float *bb, const float *bc,
                               void *y, void *ta, void *tb, const ql_epilogue *epi,
                               void *workspace, size_t workspace_bytes, void *stream);
size_t qlayer_linear_fwd_ex_workspace_size(const ql_linear_desc *desc, const ql_epilogue *epi);
ql_status qlayer_linear_fwd_ex(const ql_linear_desc *desc, const void *x,
                               const void *wa, const void *wb, const void *wc,
                               const float *ba, const float *bb, const float *bc,
                               void *y, void *ta, void *tb, const ql_epilogue *epi,
                               void *workspace, size_t workspace_bytes, void *stream);

/* ---------------------------------------------------------------------------
 * Backward behind the fused ReLU -- section 4.2, model construction (a ReLU
 * after each quadratic layer) and section 4.3 eq:SD: the layer's gradients
 * when its forward ran the epilogue's ReLU, y' = relu(Y) (ql_epilogue.relu,
 * no scale or shift).  With gy = dl/dy', G = dl/dY = gy o [y' > 0] (zero
 * where y' <= 0 or is NaN), then dX, dW_t and db_t from G exactly as
 * qlayer_conv2d_bwd_data / qlayer_conv2d_bwd_weight (qlayer_linear_bwd for
 * the dense form) compute them, bitwise.  G goes once into the front of the
 * workspace and feeds both gradients: one pass over gy and y', and no dl/dY
 * tensor of the caller.
 *   x       : the layer input (NHWC / (B,I)), required (T2, T2&4 and the
 *             weight gradient read it).
 *   gy, y_out : dl/dy' and the stored y', (N,Ho,Wo,O) / (B,O), required.
 *   ta, tb  : the saved maps of the neuron type (as the regular backward).
 *   wa, wb, wc : required when dx is requested.
 *   dx      : or NULL to skip the input gradient.
 *   dwa.. / dba.. : float32, all of the type's terms or none; db needs dW.
 *   At least one of dx / dW must be requested.  Every pointer 16-byte
 *   aligned.  Workspace: at least the query's bytes (which covers both
 *   gradients); QL_EWORKSPACE if smaller or NULL.  Validation is complete
 *   before the first launch.
 * ------------------------------------------------------------------------- */
size_t qlayer_conv2d_bwd_relu_workspace_size(const ql_conv_desc *desc);
ql_status qlayer_conv2d_bwd_relu(const ql_conv_desc *desc, const void *x, const void *gy, const void *y_out,
                                 const void *ta, const void *tb,
                                 const void *wa, const void *wb, const void *wc, void *dx,
                                 float *dwa, float *dwb, float *dwc,
                                 float *dba, float *dbb, float *dbc,
                                 void *workspace, size_t workspace_bytes, void *stream);
size_t qlayer_linear_bwd_relu_workspace_size(const ql_linear_desc *desc);
ql_status qlayer_linear_bwd_relu(const ql_linear_desc *desc, const void *x, const void *gy, const void *y_out,
                                 const void *ta, const void *tb,
                                 const void *wa, const void *wb, const void *wc, void *dx,
                                 float *dwa, float *dwb, float *dwc,
                                 float *dba, float *dbb, float *dbc,
                                 void *workspace, size_t workspace_bytes, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* QLAYER_H */
