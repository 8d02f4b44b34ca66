/*
 * bnr.h -- C ABI of libbnr: restructured batch normalisation (BN
 * Fission-n-Fusion) for CNN training on AMD Instinct MI355X (gfx950).
 *
 * The method ("Restructuring Batch Normalization to Accelerate CNN Training",
 * arXiv 1807.01702, Sec. 3.2, Fig. 5) splits each BN layer into
 *   sub-BN1: the per-channel mini-batch statistics, computed in one sweep as
 *            sum(x) and sum(x^2) (mean/variance fusion, V(X) = E(X^2) - E(X)^2)
 *            and fused into the epilogue of the CONV that produces x, and
 *   sub-BN2: (x - mean) * rstd * gamma + beta, fused with the following ReLU
 *            into the input prologue of the CONV that consumes the result;
 * and, in the backward pass, fuses the per-channel reductions sum(dy) and
 * sum(dy * xhat) into the epilogue of the backward CONV that produces dy, and
 * the input-gradient correction into the prologue of the next backward CONV.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Tensors are NHWC.  A tensor "view" is a device pointer to its first
 *   channel at pixel 0 plus a pixel stride `ldc` in elements (a view may be a
 *   channel slice of a wider buffer, e.g. a DenseNet concatenation buffer).
 *   m = n*h*w pixels.  Statistics run over all m pixels of a channel.
 * - Storage type (bnr_dtype) applies to activations, conv weights and
 *   activation gradients.  BN parameters, statistics, dgamma/dbeta and conv
 *   weight gradients are always float32.  All arithmetic accumulates in
 *   float32; cross-tile statistics combine in float64.
 * - Conv weights are [k][k][c_in][c_out] (dense, dtype); k is 1 or 3, stride
 *   1, zero padding k/2 (padding is applied to the CONV input, i.e. after BN
 *   and ReLU: padded taps contribute 0).
 * - All pointers are device pointers owned by the caller, 16-byte aligned.
 *   Channel counts, `ldc` values and channel offsets are multiples of 8 for
 *   BNR_BF16 and of 4 for BNR_F32 (one 16-byte vector).
 * - `stream` is a hipStream_t (NULL: the null stream).  Every call is
 *   asynchronous on it; errors of kernels in flight surface at the caller's
 *   next synchronisation.
 * - Every call validates all arguments before it launches anything: a status
 *   other than BNR_OK means nothing was launched and nothing was written.
 *   bnr_last_error() then describes the problem (thread-local string).
 * - Workspace: device memory the caller provides for per-tile partial sums and
 *   staging; query its size with the matching bnr_*_workspace_size call.  The
 *   library allocates no device memory of its own, with one exception: the
 *   fixed static scratch array of bnr_bn_relu_conv_fwd_static (one per GPU,
 *   held until the process ends).  Workspace contents need no initialisation
 *   and are dead after the call's kernels complete.
 * - Outputs must not alias inputs unless an entry point says otherwise.
 *   Calls keep no state between them and are thread-safe, except for the
 *   process-wide launch-timing switch of bnr_trace_begin / bnr_trace_end
 *   (a diagnostic) and the static scratch array named above.
 */
#ifndef BNR_H
#define BNR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    BNR_OK = 0,
    BNR_ERR_NULL = 1,        /* a required pointer is NULL                          */
    BNR_ERR_SHAPE = 2,       /* a size is non-positive, inconsistent or too large   */
    BNR_ERR_DTYPE = 3,       /* unknown storage type                                 */
    BNR_ERR_ALIGN = 4,       /* pointer not 16-byte aligned, or channel count / ldc  */
                             /* not a multiple of the 16-byte vector                 */
    BNR_ERR_WORKSPACE = 5,   /* workspace NULL or smaller than required              */
    BNR_ERR_UNSUPPORTED = 6, /* well-formed request outside what is implemented      */
    BNR_ERR_HIP = 7,         /* the HIP runtime rejected a launch                    */
    BNR_ERR_ALIAS = 8        /* an output overlaps an input it may not overlap       */
} bnr_status;

typedef enum { BNR_F32 = 0, BNR_BF16 = 1 } bnr_dtype;

/* One stride-1, zero-padded CONV on NHWC views. */
typedef struct {
    int32_t n, h, w;       /* batch size and image height/width; m = n*h*w        */
    int32_t c_in, c_out;   /* input / output channels                            */
    int32_t k;             /* filter size: 1 or 3 (pad k/2)                      */
    int32_t in_ldc;        /* pixel stride (elements) of the input view           */
    int32_t out_ldc;       /* pixel stride (elements) of the output view          */
    bnr_dtype dtype;       /* storage type of activations, weights, gradients    */
} bnr_conv_desc;

/* Per-channel BN state of one BN layer (float32 arrays of the BN's C channels).
 * Training-mode BN (Sec. 2.2; Sec. 3.2 for the one-sweep statistics):
 *   mean = sum(x)/m, var = sum(x^2)/m - mean^2 (biased), rstd = 1/sqrt(var+eps),
 *   y = gamma * (x - mean) * rstd + beta.
 * Statistics producers write mean/var/rstd; consumers read mean/rstd. */
typedef struct {
    const float *gamma;    /* [C] scale                                            */
    const float *beta;     /* [C] shift                                            */
    float *mean;           /* [C] mini-batch mean                                  */
    float *var;            /* [C] biased mini-batch variance (may be NULL)         */
    float *rstd;           /* [C] 1/sqrt(var + eps)                                */
    float eps;             /* > 0                                                  */
    /* Robust one-sweep statistics (optional; NULL/0 leaves every result as
     * above).  With shift K set, the one-sweep producers (statistics sweep,
     * CONV statistics epilogues, stem CONV, max pooling) accumulate
     * sum(x - K) and sum((x - K)^2) and the finalisation forms
     * mean = K + S1/m, var = S2/m - (S1/m)^2: the same values in exact
     * arithmetic (Sec. 3.2, mean/variance fusion), without the cancellation of
     * E[x^2] - E[x]^2 when |mean| >> std (K = e.g. the running mean).  The
     * two-pass (unfused) statistics ignore K.  With running_mean set the
     * finalisation also updates running_mean (and running_var, unbiased
     * m/(m-1) scaling, when set): r = (1 - momentum) r + momentum * batch
     * value.  shift may alias running_mean (read before the update). */
    const float *shift;    /* [C] or NULL                                          */
    float *running_mean;   /* [C] or NULL                                          */
    float *running_var;    /* [C] or NULL                                          */
    float momentum;        /* in [0, 1]                                            */
    /* Low part of the mean (optional).  When set, every statistics producer
     * also writes mean_lo = mean64 - mean, the float32 rounding of what the
     * float32 mean drops from the float64 value it was rounded from, and every
     * consumer of float32 data normalises the centred value x - mean with it:
     * y = (x - mean) c0 + beta - mean_lo c0 (c0 = gamma rstd), xhat and the
     * deferred input gradient alike.  The plain form x c0 + beta - mean c0
     * loses |mean| 2^-24 through the float32 mean and product, above 1e-4 of
     * the normalised value once |mean| / std reaches about 10^3; x - mean is
     * exact there (the operands are within a factor of two), so the centred
     * form keeps float32 accuracy at any offset.  bf16 consumers use mean
     * alone (the storage itself carries |x| 2^-9).  The same BN arrays must
     * reach every consumer of one tensor (forward, ReLU mask, recompute). */
    float *mean_lo;        /* [C] or NULL                                          */
} bnr_bn;

/* Where the gradient of a CONV's output comes from (backward entry points). */
typedef enum {
    BNR_GRAD_DENSE = 0,    /* g: materialised [m][c_out] view (pixel stride g_ldc)  */
    BNR_GRAD_BN = 1,       /* the CONV output is the input x of a BN whose output  */
                           /* gradient dy (after its ReLU mask) and reductions     */
                           /* dgamma = sum(dy*xhat), dbeta = sum(dy) are known:    */
                           /* g = gamma*rstd*(dy - dbeta/m - xhat*dgamma/m),       */
                           /* xhat = (x - mean)*rstd, computed on the fly (Sec.3.2 */
                           /* backward fusion); never materialised                 */
    BNR_GRAD_AVGPOOL2 = 2, /* the CONV output feeds a 2x2/2 average pooling and g  */
                           /* is the pooled gradient [n][h/2][w/2][c_out]; the     */
                           /* CONV-output gradient g[p/2]/4 is formed on the fly   */
    BNR_GRAD_SPLIT = 3     /* the CONV output x is read by several BN layers that  */
                           /* share its statistics (DenseNet concatenation, Sec.   */
                           /* 3.2 inter-composite-layer fusion) and their input    */
                           /* gradients were left in summed form by                */
                           /* bnr_bwd_fused_split: g view holds                    */
                           /* D = sum_l gamma_l*rstd*dy_l, alpha/betap the per-    */
                           /* channel sums; g = D + alpha + betap*xhat, xhat =      */
                           /* (x - mean)*rstd from bn, formed on the fly           */
} bnr_grad_kind;

typedef struct {
    bnr_grad_kind kind;
    const void *g;         /* DENSE, AVGPOOL2, SPLIT (D): gradient view             */
    int32_t g_ldc;         /* DENSE, AVGPOOL2, SPLIT: its pixel stride              */
    const void *dy;        /* BN: [m][c_out] dense gradient of the BN output        */
    const void *x;         /* BN, SPLIT: the BN input (= this CONV's output) view    */
    int32_t x_ldc;         /* BN, SPLIT: its pixel stride                            */
    const bnr_bn *bn;      /* BN: gamma, mean, rstd of that BN; SPLIT: mean, rstd    */
    const float *dgamma;   /* BN: [c_out]                                            */
    const float *dbeta;    /* BN: [c_out]                                            */
    const float *alpha;    /* SPLIT: [c_out]                                         */
    const float *betap;    /* SPLIT: [c_out]                                         */
} bnr_grad_src;

/* ------------------------------------------------------------ sizes ---- */
size_t bnr_stats_workspace_size(int64_t m, int32_t c);
/* Workspace bytes enough for every conv entry point on this descriptor. */
size_t bnr_workspace_size(const bnr_conv_desc *d);

/* ------------------------------------------------------ forward path ---- */

/* Standalone sub-BN1 (Sec. 3.2, mean/variance fusion) for a BN whose producer
 * is not a CONV (a block input, a concatenation): one read sweep of x[m][c]
 * (pixel stride ldc) accumulating sum(x), sum(x^2) per channel (float32 per
 * tile, float64 across tiles), then mean/var/rstd into bn (gamma/beta unused). */
bnr_status bnr_bn_stats(int64_t m, int32_t c, int32_t ldc, bnr_dtype dtype, const void *x,
                        bnr_bn *bn, void *ws, size_t ws_bytes, void *stream);

/* Fused CONV + sub-BN1 (Sec. 3.2, CONV1-(sub-BN1) fusion): y = conv(x, w) and,
 * in the same kernel, per-output-channel sum(y), sum(y^2) of the values as
 * stored in y; then mean/var/rstd of y into y_bn.  x is used as is (no BN
 * before this CONV). */
bnr_status bnr_conv_bn_stats_fwd(const bnr_conv_desc *d, const void *x, const void *w, void *y,
                                 bnr_bn *y_bn, void *ws, size_t ws_bytes, void *stream);

/* Fused (sub-BN2)-ReLU-CONV (Sec. 3.2): y = conv(relu(gamma*(x-mean)*rstd+beta), w)
 * with the normalisation and ReLU applied while the CONV reads x (x_bn gives
 * gamma, beta, mean, rstd of x's c_in channels).  If y_bn is not NULL the
 * epilogue also produces the statistics of y (CONV-(sub-BN1) fusion of the
 * next BN) exactly as bnr_conv_bn_stats_fwd does. */
bnr_status bnr_bn_relu_conv_fwd(const bnr_conv_desc *d, const void *x, const bnr_bn *x_bn,
                                const void *w, void *y, bnr_bn *y_bn,
                                void *ws, size_t ws_bytes, void *stream);

/* bnr_bn_relu_conv_fwd that also writes the BN+ReLU output it feeds to the
 * CONV, z = relu(gamma*(x-mean)*rstd+beta), to the view z[m][c_in] (pixel
 * stride z_ldc): the O2' sweep of the paper's fused (sub-BN2)-ReLU-CONV layer
 * (Sec. 3.2), materialised for the BN backward.  z holds exactly the values
 * the CONV multiplies (in the storage type).  The backward that reads it is
 * bnr_bwd_fused_o2; bnr_bn_relu_conv_fwd + bnr_bwd_fused is the same
 * computation with z recomputed from x instead (one sweep fewer).
 * Workspace: bnr_workspace_size(d).  Errors as bnr_bn_relu_conv_fwd, plus
 * BNR_ERR_NULL for z NULL, BNR_ERR_ALIAS if z overlaps x, y or w. */
bnr_status bnr_bn_relu_conv_fwd_o2(const bnr_conv_desc *d, const void *x, const bnr_bn *x_bn,
                                   const void *w, void *y, bnr_bn *y_bn, void *z, int32_t z_ldc,
                                   void *ws, size_t ws_bytes, void *stream);

/* DenseNet transition layer, fused (Sec. 2.3 transition layer; Sec. 3.2
 * (sub-BN2)-ReLU-CONV fusion): y = avgpool2x2(conv1x1(relu(bn(x)))) computed
 * as conv1x1(avgpool2x2(relu(bn(x)))) -- both operations are linear, so the
 * 2x2 average of the normalised, rectified input is formed while the CONV
 * reads x and the CONV runs on the n (h/2) (w/2) pooled pixels (a quarter of
 * the multiply-adds; no full-resolution output is written).  d describes the
 * full-resolution CONV (k = 1, h and w even, in_ldc: pixel stride of x);
 * y is the pooled [n][h/2][w/2][c_out] view with pixel stride d->out_ldc
 * (e.g. the first channels of the next dense block's buffer).  y_bn (may be
 * NULL): statistics of y from the epilogue.  Workspace: bnr_workspace_size(d).
 * The backward is bnr_bwd_fused / bnr_bwd_fused_split with a
 * BNR_GRAD_AVGPOOL2 gradient source (the pooled gradient formed on load).
 * Errors: BNR_ERR_UNSUPPORTED for k != 1, BNR_ERR_SHAPE for odd h or w,
 * BNR_ERR_NULL without x_bn, BNR_ERR_ALIAS if y overlaps x. */
bnr_status bnr_bn_relu_conv_pool_fwd(const bnr_conv_desc *d, const void *x, const bnr_bn *x_bn,
                                     const void *w, void *y, bnr_bn *y_bn,
                                     void *ws, size_t ws_bytes, void *stream);

/* ResNet bottleneck boundary, fused (Sec. 2.2 element-wise sum; Sec. 3.2
 * (sub-BN2)-ReLU-CONV fusion): the last BN of a block, the identity addition
 * and the ReLU run in the prologue of the next block's first 1x1 CONV:
 *   r = relu(gamma*(y-mean)*rstd + beta + ident)   (written to the view r:
 *       the next block's identity and the ReLU operand of the backward),
 *   out = conv1x1(r, w), with the statistics of out into out_bn (nullable).
 * d describes the CONV (k = 1; c_in channels of y, ident and r; in_ldc: pixel
 * stride of y; out_ldc of out).  y_bn: gamma, beta, mean, rstd of y.  r is
 * exactly what bnr_bn_add_relu_fwd would write.  Workspace:
 * bnr_workspace_size(d).  r must not overlap y, ident, w or out; out must not
 * overlap y, ident or w (BNR_ERR_ALIAS).  k != 1: BNR_ERR_UNSUPPORTED. */
bnr_status bnr_bn_add_relu_conv_fwd(const bnr_conv_desc *d, const void *y, const bnr_bn *y_bn,
                                    const void *ident, int32_t ident_ldc, void *r, int32_t r_ldc,
                                    const void *w, void *out, bnr_bn *out_bn,
                                    void *ws, size_t ws_bytes, void *stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * bnr_bn_relu_conv_fwd with the same arguments and results, but no workspace
 * argument.  Its workspace is a static __device__ array of 16 MiB per GPU
 * (allocated with the library's code object, held until the process ends);
 * the call itself allocates nothing and creates no HIP events.
 *   Limit: a CONV whose forward workspace (packed weights, statistics partial
 *   rows, combine stage) exceeds 16 MiB returns BNR_ERR_WORKSPACE before any
 *   launch.  Every layer of the dense block, the ResNet stack and DenseNet-121
 *   at the shapes of this library's workloads fits.
 *   Calls on one GPU share that GPU's array and leave their partial sums in
 *   it: two calls whose kernels overlap in time on one GPU (different
 *   streams, different host threads) race; serialise them on one stream.
 *   No part of the array needs to start at zero.
 *   The first call on each GPU looks up the array's device address on that
 *   GPU (hipGetSymbolAddress) with the GPU current. */
bnr_status bnr_bn_relu_conv_fwd_static(const bnr_conv_desc *d, const void *x, const bnr_bn *x_bn,
                                       const void *w, void *y, bnr_bn *y_bn, void *stream);

/* 2x2 average pooling, stride 2, of x[n][h][w][c] (pixel stride ldc) into the
 * view y[n][h/2][w/2][c] (pixel stride y_ldc, e.g. the first channels of the
 * next dense block's concatenation buffer); h and w even.  (DenseNet
 * transition layer, Sec. 2.3.) */
bnr_status bnr_avgpool2_fwd(int32_t n, int32_t h, int32_t w, int32_t c, bnr_dtype dtype,
                            const void *x, int32_t ldc, void *y, int32_t y_ldc, void *stream);

/* ----------------------------------------------------- backward path ---- */

/* Backward of bnr_avgpool2_fwd as a separate sweep (used by the unfused
 * path): gx[n][y][x][c] = g[n][y/2][x/2][c] / 4, written to the view gx
 * (pixel stride gx_ldc) from the pooled gradient view g (pixel stride g_ldc). */
bnr_status bnr_avgpool2_bwd(int32_t n, int32_t h, int32_t w, int32_t c, bnr_dtype dtype, const void *g,
                            int32_t g_ldc, void *gx, int32_t gx_ldc, void *stream);

/* Backward of one BN-ReLU-CONV chain (or of a plain CONV when x_bn is NULL),
 * with the paper's backward fission/fusion (Sec. 3.2, Fig. 5b):
 *   1. dgrad: dz = conv_transpose(g, w), g from *g_src (prologue);
 *      epilogue (x_bn != NULL): recompute y = gamma*xhat+beta from x, apply the
 *      ReLU mask dy = dz*[y>0], store dy[m][c_in] (dense), and accumulate
 *      per-channel sum(dy), sum(dy*xhat) over the tile;
 *   2. combine the tiles: dbeta = sum(dy), dgamma = sum(dy*xhat)   (x_bn != NULL);
 *   3. wgrad: dw = sum over pixels of relu(bn(x)) (x itself if x_bn is NULL),
 *      recomputed from x in the prologue, times g;
 *   4. optional standalone input gradient: if dx != NULL, the BN input gradient
 *      gamma*rstd*(dy - dbeta/m - xhat*dgamma/m) (x_bn != NULL) or dz itself
 *      (x_bn == NULL) is written to (dx_accumulate = 0) or added to
 *      (dx_accumulate = 1) the view dx (pixel stride dx_ldc).  dx may alias x
 *      only if x_bn is NULL and never otherwise; with dx_accumulate = 1 the old
 *      contents of dx are read.  When dx is NULL the BN input gradient stays
 *      deferred: a later call consumes it as BNR_GRAD_BN from (dy, x, dgamma,
 *      dbeta).
 * Outputs: dw [k][k][c_in][c_out] float32 (overwritten); dgamma, dbeta [c_in]
 * float32 and dy (required when x_bn != NULL). */
bnr_status bnr_bwd_fused(const bnr_conv_desc *d, const void *x, const bnr_bn *x_bn, const void *w,
                         const bnr_grad_src *g_src, float *dw, float *dgamma, float *dbeta, void *dy,
                         void *dx, int32_t dx_ldc, int32_t dx_accumulate,
                         void *ws, size_t ws_bytes, void *stream);

/* bnr_bwd_fused for a forward run by bnr_bn_relu_conv_fwd_o2 (the paper's
 * O2' structure, Sec. 3.2): z is that forward's stored BN+ReLU output (view
 * [m][c_in], pixel stride z_ldc).  Step 1's epilogue reads z in place of x:
 * dy = dz*[z>0] and xhat = (z - beta)/gamma wherever dy can be non-zero (so
 * z's rounding enters dgamma through xhat); a thread whose 16-byte channel
 * vector holds a channel with gamma = 0 (xhat not recoverable from z) reads x
 * there instead, with the formulas of bnr_bwd_fused.  Step 3 multiplies z as
 * it is (no recompute).  Step 4 and the outputs are those of bnr_bwd_fused
 * (x is still the BN input).  Errors as bnr_bwd_fused, plus BNR_ERR_NULL for
 * x_bn or z NULL and BNR_ERR_ALIAS if z overlaps dy or dx. */
bnr_status bnr_bwd_fused_o2(const bnr_conv_desc *d, const void *x, const bnr_bn *x_bn, const void *z,
                            int32_t z_ldc, const void *w, const bnr_grad_src *g_src, float *dw, float *dgamma,
                            float *dbeta, void *dy, void *dx, int32_t dx_ldc, int32_t dx_accumulate,
                            void *ws, size_t ws_bytes, void *stream);

/* The two independent halves of bnr_bwd_fused (and of bnr_bwd_fused_split
 * below), for callers that overlap a layer's weight gradient with the data
 * gradients of the layers before it (e.g. on a second stream).  Step 3 reads
 * only x, x_bn and what g_src reads -- nothing steps 1-2 write -- so the
 * halves may run in either order or concurrently once g_src is complete.
 *   bnr_bwd_data:    steps 1, 2 and 4 of bnr_bwd_fused (all its arguments but dw);
 *   bnr_bwd_weights: step 3 (dw [k][k][c_in][c_out] float32, overwritten; x_bn
 *                    NULL: the CONV input is x itself).
 * Each call needs its own workspace while another call may be in flight. */
bnr_status bnr_bwd_data(const bnr_conv_desc *d, const void *x, const bnr_bn *x_bn, const void *w,
                        const bnr_grad_src *g_src, float *dgamma, float *dbeta, void *dy,
                        void *dx, int32_t dx_ldc, int32_t dx_accumulate,
                        void *ws, size_t ws_bytes, void *stream);
bnr_status bnr_bwd_weights(const bnr_conv_desc *d, const void *x, const bnr_bn *x_bn,
                           const bnr_grad_src *g_src, float *dw, void *ws, size_t ws_bytes, void *stream);

/* Standalone BN input gradient for a BN whose producer is not a CONV (block
 * input, concatenation): dx = gamma*rstd*(dy - dbeta/m - xhat*dgamma/m) from
 * dy[m][c] (dense), x (pixel stride x_ldc), written or added into dx (pixel
 * stride dx_ldc).  dx may alias dy's storage only if dx_accumulate = 0 and the
 * views coincide exactly. */
bnr_status bnr_bn_dx(int64_t m, int32_t c, bnr_dtype dtype, const void *dy, const void *x, int32_t x_ldc,
                     const bnr_bn *bn, const float *dgamma, const float *dbeta,
                     void *dx, int32_t dx_ldc, int32_t dx_accumulate, void *stream);

/* ------------------------- concatenation BNs (DenseNet, ICF) ---------- */

/* Inter-composite-layer fusion (Sec. 3.2, last paragraph; the paper leaves it
 * to future work and estimates its gain in Sec. 5).  In a dense block every
 * BN1 reads channels of one concatenation buffer, and all BN layers that read
 * a channel see the same values, hence the same mini-batch mean and rstd.
 * Forward: each channel's statistics are produced once, by the epilogue of the
 * CONV that writes it (bnr_bn_relu_conv_fwd with y_bn viewing the shared
 * per-channel arrays at the channel offset) or by one bnr_bn_stats sweep over
 * the block input; every BN1 then reads them, so no BN1 sweeps its input.
 * Backward: the input gradient of channel c summed over its BN consumers l is
 *   sum_l gamma_l*rstd*(dy_l - dbeta_l/m - xhat*dgamma_l/m)
 *     = D + alpha + betap*xhat,  D = sum_l gamma_l*rstd*dy_l,
 *   alpha = -sum_l gamma_l*rstd*dbeta_l/m,  betap = -sum_l gamma_l*rstd*dgamma_l/m,
 * so each consumer's backward adds its term to D in its data-gradient
 * epilogue and to alpha/betap in its reductions combine, and the producer's
 * backward forms the gradient on load (BNR_GRAD_SPLIT).  (This factorisation
 * is this library's reading of the fused Split-layer backward.) */

/* bnr_bwd_fused for a BN whose input x is a concatenation slice: the same
 * steps 1-3 (dgrad with the BN-backward epilogue, dbeta/dgamma combine,
 * wgrad), except that the epilogue does not store dy but writes
 * (accumulate = 0) or adds (accumulate = 1) gamma*rstd*dy into the view gsum
 * (D above; [m][c_in], pixel stride gsum_ldc), and the combine also writes or
 * adds alpha and betap ([c_in] float32).  x_bn is required.  gsum must not
 * overlap x or any view g_src reads; with accumulate = 1 its old contents are
 * read.  Outputs: dw, dgamma, dbeta (overwritten), gsum, alpha, betap. */
bnr_status bnr_bwd_fused_split(const bnr_conv_desc *d, const void *x, const bnr_bn *x_bn, const void *w,
                               const bnr_grad_src *g_src, float *dw, float *dgamma, float *dbeta,
                               void *gsum, int32_t gsum_ldc, int32_t accumulate, float *alpha, float *betap,
                               void *ws, size_t ws_bytes, void *stream);

/* Steps 1-2 of bnr_bwd_fused_split (its arguments but dw); its weight
 * gradient is bnr_bwd_weights on the same descriptor, x, x_bn and g_src. */
bnr_status bnr_bwd_data_split(const bnr_conv_desc *d, const void *x, const bnr_bn *x_bn, const void *w,
                              const bnr_grad_src *g_src, float *dgamma, float *dbeta,
                              void *gsum, int32_t gsum_ldc, int32_t accumulate, float *alpha, float *betap,
                              void *ws, size_t ws_bytes, void *stream);

/* Materialise a summed BN input gradient: dx = gsum + alpha + betap*xhat with
 * xhat = (x - mean)*rstd (mean, rstd from bn), written to (dx_accumulate = 0)
 * or added into (1) the view dx.  All views [m][c] with their pixel strides.
 * dx may alias gsum only if the views coincide exactly and dx_accumulate = 0;
 * dx must not overlap x. */
bnr_status bnr_split_dx(int64_t m, int32_t c, bnr_dtype dtype, const void *gsum, int32_t gsum_ldc,
                        const void *x, int32_t x_ldc, const bnr_bn *bn, const float *alpha, const float *betap,
                        void *dx, int32_t dx_ldc, int32_t dx_accumulate, void *stream);

/* ------------------------------------------------- unfused A/B path ---- */

typedef enum {
    BNR_MODE_BASELINE = 0, /* the paper's unfused layer chain (Sec. 3.2, upper half  */
                           /* of Fig. 5): mean sweep, variance sweep, normalise      */
                           /* (write y), ReLU (read y, write z), CONV (read z);      */
                           /* backward: CONV dgrad (write dz) and wgrad (read z),    */
                           /* ReLU backward (write dy), BN reductions sweep, BN      */
                           /* input-gradient sweep (write dx)                        */
    BNR_MODE_RCF = 1,      /* ReLU-CONV fusion only (Sec. 3.2): ReLU applied while   */
                           /* the CONV reads y; mask applied in the dgrad epilogue    */
    BNR_MODE_RCF_MVF = 2   /* RCF plus one-sweep mean/variance statistics            */
} bnr_ref_mode;

typedef struct {
    const void *x;         /* BN input view, pixel stride desc.in_ldc               */
    bnr_bn *bn;            /* gamma, beta in; mean, var, rstd written by forward    */
    const void *w;         /* CONV weights                                          */
    void *y;               /* [m][c_in] dense: BN output (materialised)             */
    void *z;               /* [m][c_in] dense: ReLU output (BASELINE only)          */
    void *out;             /* CONV output view, pixel stride desc.out_ldc           */
    const void *g;         /* backward: gradient of out, [m][c_out], stride g_ldc   */
    int32_t g_ldc;
    void *dz;              /* backward: [m][c_in] CONV input gradient (BASELINE)    */
    void *dy;              /* backward: [m][c_in] BN output gradient                */
    float *dw, *dgamma, *dbeta;
    void *dx;              /* backward: BN input gradient view, stride dx_ldc       */
    int32_t dx_ldc;
    int32_t dx_accumulate;
} bnr_ref_args;

/* The same training math as the fused entry points through separate,
 * unfused kernels (same GEMM core with fusion switched off), for A/B
 * comparison of time and HBM traffic.  backward = 0: forward of one
 * BN-ReLU-CONV chain; backward = 1: its backward. */
bnr_status bnr_reference_path(bnr_ref_mode mode, int32_t backward, const bnr_conv_desc *d,
                              const bnr_ref_args *a, void *ws, size_t ws_bytes, void *stream);

/* ------------------------------------------ residual blocks (ResNet) ---- */

/* Plain CONV forward y = conv(x, w) (no BN work): a CONV whose input has no
 * BN in front of it and whose output statistics are not needed, e.g. the
 * first CONV of a block in the unfused A/B chain. */
bnr_status bnr_conv_fwd(const bnr_conv_desc *d, const void *x, const void *w, void *y, void *ws, size_t ws_bytes,
                        void *stream);

/* Residual-block tail out = relu(gamma*(y-mean)*rstd + beta + id) in one
 * element-wise sweep ([m][c] views; bn holds the statistics of y, already
 * produced by the CONV that wrote y).  The BN here is followed by an addition
 * and a ReLU rather than by a CONV, so sub-BN2 cannot be fused into a
 * following CONV prologue (Sec. 3.2 fuses sub-BN2 only into a following
 * CONV); it runs as a standalone pass.  out may alias id exactly. */
bnr_status bnr_bn_add_relu_fwd(int64_t m, int32_t c, bnr_dtype dtype, const void *y, int32_t y_ldc,
                               const bnr_bn *bn, const void *id, int32_t id_ldc, void *out, int32_t out_ldc,
                               void *stream);

/* Backward of bnr_bn_add_relu_fwd up to the BN reductions, in one sweep:
 * gm = g * [out > 0] (the gradient of the identity input and of the BN
 * output), dbeta = sum(gm), dgamma = sum(gm * xhat) with xhat from y and bn
 * (the standard BN gradients).  The BN input gradient is not formed: the
 * CONV that produced y consumes it deferred (BNR_GRAD_BN with dy = gm).  gm
 * may alias g exactly.  ws: bnr_stats_workspace_size(m, c) bytes. */
bnr_status bnr_bn_add_relu_bwd(int64_t m, int32_t c, bnr_dtype dtype, const void *g, int32_t g_ldc,
                               const void *out, int32_t out_ldc, const void *y, int32_t y_ldc, const bnr_bn *bn,
                               void *gm, int32_t gm_ldc, float *dgamma, float *dbeta, void *ws, size_t ws_bytes,
                               void *stream);

/* Unfused A/B counterpart of the two calls above (the reference layer
 * chain): forward, two-pass statistics of y into bn (mean, var, rstd), a
 * normalise sweep (write tmp, dense [m][c]) and an add + ReLU sweep (write
 * out); backward, a ReLU-backward sweep (write gm, dense), a reductions sweep
 * (dgamma, dbeta) and an input-gradient sweep (write dx). */
typedef struct {
    const void *y;       /* BN input                                      */
    int32_t y_ldc;
    bnr_bn *bn;
    const void *id;      /* forward: identity input                       */
    int32_t id_ldc;
    void *out;           /* forward: output; backward: the forward output */
    int32_t out_ldc;
    void *tmp;           /* forward scratch, dense [m][c]                 */
    const void *g;       /* backward: gradient of out                     */
    int32_t g_ldc;
    void *gm;            /* backward: masked gradient, dense [m][c]       */
    float *dgamma, *dbeta;
    void *dx;            /* backward: BN input gradient                   */
    int32_t dx_ldc;
} bnr_addrelu_ref_args;
bnr_status bnr_reference_bn_add_relu(int32_t backward, int64_t m, int32_t c, bnr_dtype dtype,
                                     const bnr_addrelu_ref_args *a, void *ws, size_t ws_bytes, void *stream);

/* ------------------------------------ network ends (whole DenseNet) ---- */

/* The first CONV of the network: 7x7, stride 2, zero padding 3 (Sec. 3.1
 * notes DenseNet-121's first CONV is 7x7), c_in image channels -> 64.
 *   img [n][h][w][4] (dtype): channels 0..c_in-1 are used, the rest are read
 *       as 0 (one 8-byte bf16 / 16-byte float32 pixel);  w <= 256.
 *   w   [7][7][c_in][64] (dtype).
 *   s   [n][ho][wo][64] dense output, ho = (h-1)/2 + 1, wo = (w-1)/2 + 1. */
typedef struct {
    int32_t n, h, w;       /* batch size, image height and width                 */
    int32_t c_in;          /* image channels, 1..4                               */
    bnr_dtype dtype;
} bnr_stem_desc;

/* Workspace bytes for bnr_stem_conv_fwd and bnr_stem_wgrad on d. */
size_t bnr_stem_workspace_size(const bnr_stem_desc *d);

/* First CONV with the sub-BN1 statistics epilogue of the BN after it (Sec.
 * 3.2 CONV-(sub-BN1) fusion): s = conv(img, w) and, when s_bn is not NULL,
 * the mean/var/rstd of s's 64 channels (float32 per-workgroup sums of the
 * stored values, float64 combine) into s_bn.  (The float32 storage type runs
 * a direct CONV and a statistics sweep: it is the parity configuration.) */
bnr_status bnr_stem_conv_fwd(const bnr_stem_desc *d, const void *img, const void *w, void *s,
                             bnr_bn *s_bn, void *ws, size_t ws_bytes, void *stream);

/* Weight gradient of the first CONV: dw[7][7][c_in][64] (float32, overwritten)
 * = sum over output pixels of the image patch times g, g the gradient of s
 * from g_src: BNR_GRAD_DENSE (view g, pixel stride g_ldc) or BNR_GRAD_BN (the
 * BN after the CONV: g = gamma*rstd*(dy - dbeta/m - xhat*dgamma/m) formed on
 * load from dy [m][64] dense and x = s, Sec. 3.2 backward fusion; rounded to
 * the storage type before the product as a stored gradient would be).  The
 * image needs no gradient. */
bnr_status bnr_stem_wgrad(const bnr_stem_desc *d, const void *img, const bnr_grad_src *g_src, float *dw,
                          void *ws, size_t ws_bytes, void *stream);

/* Workspace bytes for the two max-pooling calls below on x[n][h][w][c]. */
size_t bnr_pool_workspace_size(int32_t n, int32_t h, int32_t w, int32_t c);

/* BN -> ReLU -> 3x3 / stride 2 / pad 1 max pooling (the layer after the first
 * CONV; padded taps never win), with sub-BN2 + ReLU applied while the pooling
 * reads x (Sec. 3.2 places sub-BN2 and ReLU in the reader of the BN output):
 * y[n][ho][wo][c] = max over the window of relu(gamma*(x-mean)*rstd + beta)
 * (x_bn: gamma, beta, mean, rstd of x), or of x itself when x_bn is NULL.
 * When y_bn is not NULL the statistics of y (as stored) go to y_bn in the
 * same pass (the sub-BN1 of the next BN: a dense block's input).  Views x
 * (pixel stride x_ldc), y (pixel stride y_ldc); ho = (h-1)/2+1, wo likewise.
 * ws: bnr_pool_workspace_size bytes (may be NULL when y_bn is NULL). */
bnr_status bnr_bn_relu_maxpool_fwd(int32_t n, int32_t h, int32_t w, int32_t c, bnr_dtype dtype,
                                   const void *x, int32_t x_ldc, const bnr_bn *x_bn, void *y, int32_t y_ldc,
                                   bnr_bn *y_bn, void *ws, size_t ws_bytes, void *stream);

/* Backward of bnr_bn_relu_maxpool_fwd: each gradient gy[n][oh][ow][c] (view,
 * pixel stride gy_ldc) goes to the first maximum of its window (row-major
 * tap order).  With x_bn: the ReLU mask is applied (dy = dz [y > 0], y
 * recomputed from x), dy is stored to dy [n*h*w][c] (dense) and the BN
 * reductions dbeta = sum(dy), dgamma = sum(dy*xhat) of the stored dy are
 * written (Sec. 3.2 backward fusion); the BN input gradient stays deferred
 * (the first CONV's weight gradient consumes it as BNR_GRAD_BN).  Without
 * x_bn: dy receives the pooling input gradient.  c <= 64 with a power-of-two
 * number of 16-byte vectors; wo <= 64.  ws: bnr_pool_workspace_size bytes
 * (may be NULL without x_bn). */
bnr_status bnr_maxpool_bn_bwd(int32_t n, int32_t h, int32_t w, int32_t c, bnr_dtype dtype, const void *x,
                              int32_t x_ldc, const bnr_bn *x_bn, const void *gy, int32_t gy_ldc, void *dy,
                              float *dgamma, float *dbeta, void *ws, size_t ws_bytes, void *stream);

/* Workspace bytes for bnr_head_bwd on x[n][h][w][c]. */
size_t bnr_head_workspace_size(int32_t n, int32_t h, int32_t w, int32_t c);

/* Classifier head (the network's one FC layer, Sec. 2.2): BN -> ReLU ->
 * global average pooling -> FC -> softmax cross-entropy over the batch.
 *   x [n*h*w][c] view (pixel stride x_ldc) with its BN x_bn (gamma, beta and
 *   the statistics of x, already produced); wfc [c][classes] (dtype);
 *   bfc [classes]; labels [n] int32 (device; a label outside [0, classes)
 *   makes the loss NaN).  Outputs (float32, device): f [n][c] pooled
 *   features, logits [n][classes], dlogits = (softmax - onehot)/n, and
 *   loss [1 + n]: loss[1 + r] = -log softmax(logits[r])[label[r]] and
 *   loss[0] their mean over the batch. */
bnr_status bnr_head_fwd(int32_t n, int32_t h, int32_t w, int32_t c, int32_t classes, bnr_dtype dtype,
                        const void *x, int32_t x_ldc, const bnr_bn *x_bn, const void *wfc, const float *bfc,
                        const int32_t *labels, float *f, float *logits, float *dlogits, float *loss,
                        void *stream);

/* Backward of bnr_head_fwd from its dlogits: df = dlogits wfc^T [n][c],
 * dwfc = f^T dlogits [c][classes], dbfc = column sums [classes] (all float32,
 * overwritten), and the head BN's backward: dy = [y > 0] df/(h*w) (not
 * stored), dbeta = sum(dy), dgamma = sum(dy*xhat).  The BN input gradient:
 *   alpha, betap not NULL (x is a DenseNet concatenation, Sec. 3.2 ICF): gx
 *     receives gamma*rstd*dy and alpha/betap are written, the summed form of
 *     bnr_bwd_fused_split (accumulate = 0);
 *   alpha, betap NULL: gx receives gamma*rstd*(dy - dbeta/m - xhat*dgamma/m).
 * gx: view (pixel stride gx_ldc), must not overlap x. */
bnr_status bnr_head_bwd(int32_t n, int32_t h, int32_t w, int32_t c, int32_t classes, bnr_dtype dtype,
                        const void *x, int32_t x_ldc, const bnr_bn *x_bn, const void *wfc, const float *f,
                        const float *dlogits, float *df, float *dwfc, float *dbfc, float *dgamma, float *dbeta,
                        void *gx, int32_t gx_ldc, float *alpha, float *betap, void *ws, size_t ws_bytes,
                        void *stream);

/* Unfused A/B counterpart of a BN -> ReLU pair whose reader is not a CONV
 * (the max pooling after the first CONV): forward, two-pass statistics of
 * x[m][c] (pixel stride x_ldc) into bn (mean, var, rstd), a normalise sweep
 * (write y, dense [m][c]) and a ReLU sweep (write z, dense); backward, a
 * ReLU-backward sweep dy = gz [y > 0] (write dy, dense), a reductions sweep
 * (dgamma, dbeta) and an input-gradient sweep (write dx, pixel stride
 * dx_ldc).  ws: bnr_stats_workspace_size(m, c) bytes. */
typedef struct {
    const void *x;       /* BN input                                      */
    int32_t x_ldc;
    bnr_bn *bn;
    void *y;             /* BN output, dense [m][c] (written forward)     */
    void *z;             /* forward: ReLU output, dense [m][c]            */
    const void *gz;      /* backward: gradient of z                       */
    int32_t gz_ldc;
    void *dy;            /* backward: masked gradient, dense [m][c]       */
    float *dgamma, *dbeta;
    void *dx;            /* backward: BN input gradient                   */
    int32_t dx_ldc;
} bnr_bnrelu_ref_args;
bnr_status bnr_reference_bn_relu(int32_t backward, int64_t m, int32_t c, bnr_dtype dtype,
                                 const bnr_bnrelu_ref_args *a, void *ws, size_t ws_bytes, void *stream);

/* ------------------------------------------------------ diagnostics ---- */

/* Plain device-to-device copy of `bytes` (multiple of 16) with the same
 * streaming kernel style as the BN sweeps: the HBM-traffic calibration
 * reference for profiler byte counters. */
bnr_status bnr_hbm_copy(const void *src, void *dst, size_t bytes, void *stream);

/* Launch timing (diagnostic).  Between bnr_trace_begin and bnr_trace_end,
 * every launch of a kernel whose class is in `kernel_classes` (bit mask:
 * 1 implicit-GEMM CONV, 2 weight gradient, 4 BN sweeps and element-wise
 * passes, 8 combines / weight packing / split-K sums), up to `capacity`
 * launches, is bracketed by two HIP events recorded on the launch's own
 * stream.  bnr_trace_end waits for those events and fills, per launch, the
 * duration in ms, the algorithmic HBM bytes (each input tensor read once, each
 * output written once), the floating-point operations and a kernel id
 * (1 CONV 1x1, 2 CONV 3x3, 3 weight gradient 1x1, 4 weight gradient 3x3,
 * 5 statistics sweep, 6 element-wise pass, 7 statistics combine, 8 weight
 * packing, 9 split-K sum, 10 pooling, 11 copy, 12 first CONV, 13 first-CONV
 * weight gradient, 14 max pooling, 15 classifier head); it returns the number of
 * launches written.  Not meant for graph capture. */
bnr_status bnr_trace_begin(int32_t kernel_classes, int32_t capacity);
int32_t bnr_trace_end(double *ms, double *bytes, double *flops, int32_t *kernel_id, int32_t capacity);

const char *bnr_status_string(bnr_status s);
const char *bnr_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* BNR_H */
