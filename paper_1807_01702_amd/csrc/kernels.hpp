// kernels.hpp -- launcher interfaces between the C ABI (api.hip) and the
// HIP kernels.  Launchers assume validated arguments.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bnr {

// k_stats_partial modes
enum { ST_SUMSQ = 0, ST_SUM = 1, ST_SQDEV = 2, ST_DYX = 3 };
// k_stats_finalize modes
enum { FIN_MVF = 0, FIN_MEAN = 1, FIN_VAR = 2, FIN_BWD = 3 };
// k_elementwise modes
enum { EW_DX = 0, EW_APPLY = 1, EW_RELU = 2, EW_RELUBWD = 3, EW_BNADDRELU = 4, EW_ADDRELU = 5, EW_SPLITDX = 6 };

// Summed-gradient terms a FIN_BWD combine also writes (or adds to) for a BN
// whose input channels have several BN consumers with shared statistics:
//   alpha[c] = -gamma[c] rstd[c] dbeta[c] / m,  betap[c] = -gamma[c] rstd[c] dgamma[c] / m.
struct SplitTerms {
    const float *gamma, *rstd;
    float *alpha, *betap;         // NULL: none
    int accumulate;
    // forward finalisation (FIN_MVF, FIN_VAR): the one-sweep sums were taken
    // around shift (NULL: 0; FIN_MVF only) and the running statistics are
    // updated when rmean is set (rvar: unbiased variance)
    const float *shift;
    float *rmean, *rvar;
    float momentum;
    // FIN_MVF, FIN_MEAN: also write the low part of the float64 mean,
    // mean64 - (float)mean64 (float32 consumers centre x on the float32 mean
    // and are given this as the mean relative to it)
    float *mean_lo;
};

// Reduction scratch ("red") of a statistics combine: the float64 level-1
// sums [RS][2][C] (RS <= kRedMaxRS row splits).
constexpr int kRedMaxRS = 32;
// Up to this many partial rows the combine runs as one kernel.
constexpr int64_t kCombineOneMaxRows = 1024;
inline size_t stats_red_bytes(int C) { return (size_t)kRedMaxRS * 2 * C * sizeof(double); }
int stats_combine_splits(int64_t R);
hipError_t launch_stats_partial(int dtype, const void *x, int64_t ldc, int64_t m, int C, int mode,
                                const float *mean, const float *rstd, const void *dy, int64_t dy_ldc,
                                float *part, int64_t R, hipStream_t s, const float *ctr = nullptr);
hipError_t launch_stats_finalize(const float *part, int64_t R, int C, int64_t m, int mode, float eps, float *mean,
                                 float *var, float *rstd, float *dbeta, float *dgamma, void *red, hipStream_t s,
                                 const SplitTerms *split = nullptr);
hipError_t launch_elementwise(int dtype, int mode, int64_t m, int C, const void *x, int64_t x_ldc, const void *x2,
                              int64_t x2_ldc, const float *gamma, const float *beta, const float *mean,
                              const float *rstd, const float *dgamma, const float *dbeta, void *out,
                              int64_t out_ldc, int accumulate, hipStream_t s, const float *ctr = nullptr);
// Residual-block backward sweep: gm = g * [out > 0], per-channel sum(gm) and
// sum(gm * (y - mean) * rstd) partials [R][2][C].
// ctr (the statistics sweep's ST_DYX, the elementwise BN modes, this sweep):
// the float32 centre of the BN input (NULL: 0), mean given relative to it
// (bn_centre).
hipError_t launch_addrelu_bwd(int dtype, int64_t m, int C, const void *g, int64_t g_ldc, const void *out,
                              int64_t out_ldc, const void *y, int64_t y_ldc, const float *mean, const float *rstd,
                              void *gm, int64_t gm_ldc, float *part, int64_t R, hipStream_t s,
                              const float *ctr = nullptr);
hipError_t launch_avgpool2(int dtype, int n, int h, int w, int C, const void *x, int64_t ldc, void *y, int64_t y_ldc,
                           hipStream_t s);
hipError_t launch_avgpool2_bwd(int dtype, int n, int h, int w, int C, const void *g, int64_t g_ldc, void *gx,
                               int64_t ldc, hipStream_t s);
hipError_t launch_copy16(const void *src, void *dst, int64_t nvec, hipStream_t s);
// Split-K sum scratch: up to 8 level-1 float32 rows of len.
inline size_t sum_partials_red_bytes(int64_t len) { return 8 * (size_t)len * 4; }
int sum_partials_groups(int64_t S);
// The tail of a fused backward CONV call in one launch: dw = sum of the S
// split-K partial tiles (single level, deterministic) and the FIN_BWD combine
// of R <= kCombineOneMaxRows BN-backward partial rows (dbeta, dgamma, and the
// summed-gradient terms of split).
hipError_t launch_bwd_tail(const float *wpart, int64_t S, int64_t len, float *dw, const float *spart, int64_t R,
                           int C, int64_t m, float *dbeta, float *dgamma, const SplitTerms *split, hipStream_t s);
hipError_t launch_sum_partials(const float *part, int64_t S, int64_t len, float *out, void *red, hipStream_t s);

// ---- implicit-GEMM CONV over pixel rows (forward / data gradient) ---------
// PRO_BNRELU_POOL: the GEMM rows are the 2x2 windows of the input image (h, w
// even; m = n h w / 4 rows); a row is the average of relu(bn(x)) over its
// window's four pixels (BN, ReLU and the transition's average pooling applied
// before the linear 1x1 CONV)
// PRO_BNADDRELU: a = max(gamma (x - mean) rstd + beta + r0, 0) with x the
// residual branch's last CONV output and r0 (a2) the block's identity input;
// a is also stored to the side view (the next block's identity and the
// backward's ReLU operand)
enum { PRO_NONE = 0, PRO_BNRELU = 1, PRO_BNGRAD = 2, PRO_POOLUP = 3, PRO_RELU = 4, PRO_BNRELU_POOL = 5,
       PRO_BNADDRELU = 6 };
enum { EPI_STORE = 0, EPI_STATS = 1, EPI_BNBWD = 2, EPI_RELUMASK = 3 };
// Compile-time epilogue kinds of the persistent CONV kernels (EPI_STORE splits
// into plain store and read-add-store).
// EK_BNBWD_SC / EK_BNBWD_SCACC: the BN-backward epilogue storing (adding)
// gamma*rstd*dy instead of dy (summed-gradient form, RowsParams::e_scale).
enum { EK_STORE = 0, EK_STORE_ACC = 1, EK_STATS = 2, EK_RELUMASK = 3, EK_BNBWD = 4, EK_BNBWD_SC = 5,
       EK_BNBWD_SCACC = 6 };
inline int epilogue_kind(int epi, int accumulate, int scale) {
    if (epi == EPI_BNBWD) return scale ? (accumulate ? EK_BNBWD_SCACC : EK_BNBWD_SC) : EK_BNBWD;
    return epi == EPI_STORE ? (accumulate ? EK_STORE_ACC : EK_STORE) : (epi == EPI_STATS ? EK_STATS : EK_RELUMASK);
}

struct RowsParams {
    int dtype, taps, n, h, w;
    int64_t m;
    int K, N;                     // GEMM reduction channels (A channels), output channels
    int pro;
    const void *a;                // A source: conv input / dy (BNGRAD) / pooled gradient (POOLUP)
    int64_t a_ldc;
    const void *a2;               // BNGRAD: the BN input x (same pixels, K channels)
    int64_t a2_ldc;
    const float *p_gamma, *p_beta, *p_mean, *p_rstd, *p_dgamma, *p_dbeta;
    int p_split;                  // PRO_BNGRAD: 1 = summed gradient of several BNs (deferred_coef)
    const float *p_alpha, *p_betap;
    const float *p_ctr;           // float32 centre of the prologue BN's input (NULL: 0; p_mean relative to it)
    const void *wpack;            // weights packed by launch_pack_weights (conv_rows)
    const void *wraw;             // weights in their [k][k][c_in][c_out] layout (persistent kernels)
    int wtrans;                   // 1: data-gradient operand (GEMM K = c_out, N = c_in)
    int epi;
    void *y;                      // output view (EPI_BNBWD: dy)
    int64_t y_ldc;
    int accumulate;               // EPI_STORE; EPI_BNBWD with e_scale: add to y's old contents
    int e_scale;                  // EPI_BNBWD: y receives gamma*rstd*dy (the summed-gradient term)
    float *part;                  // EPI_STATS / EPI_BNBWD: [mtiles][2][N]
    const void *ex;               // EPI_BNBWD: BN input (N channels); EPI_RELUMASK: ReLU input
    int64_t ex_ldc;
    const float *e_gamma, *e_beta, *e_mean, *e_rstd;
    const float *e_ctr;           // EPI_BNBWD: float32 centre of ex (NULL: 0; e_mean relative to it)
    int e_zsrc;                   // EPI_BNBWD: ex is the stored z = relu(y) of the forward (O2'): mask
                                  // [z > 0], xhat = (z - beta) / gamma; channel vectors holding a
                                  // gamma = 0 channel read ex2 (the BN input x) instead
    const void *ex2;              // e_zsrc: the BN input x (N channels)
    int64_t ex2_ldc;
    const float *e_shift;         // EPI_STATS: the sums are of (y - e_shift) (NULL: 0)
    void *side;                   // PRO_BNADDRELU, PRO_BNRELU (forward, optional): the transformed
                                  // A rows are stored here too
    int64_t side_ldc;
    int buf32;                    // tiled 1x1 kernel: operand spans below 2^31 bytes (set by its launcher)
    int wdirect;                  // tiled bf16 1x1 kernel: weights read from wraw ([k][n], wtrans: [n][k]), no packing
};
int64_t rows_mtiles(int dtype, int taps, int64_t m, int n_out);
size_t rows_pack_bytes(int dtype, int taps, int K, int N);
// transpose = 0: forward packing of W[kh][kw][ci][co] (GEMM K = ci, N = co);
// transpose = 1: data-gradient packing, flipped taps, GEMM K = co, N = ci.
bool rows_direct_weights(int dtype, int taps, int64_t m, int K, int N, int64_t a_ldc, int64_t a2_ldc, int pro,
                         bool side);
hipError_t launch_pack_weights(int dtype, const void *w, int k, int c_in, int c_out, int transpose, void *wpack,
                               hipStream_t s);
hipError_t launch_conv_rows(const RowsParams &p, hipStream_t s);

// ---- persistent 1x1 CONV (weights resident in LDS, one workgroup per CU) ----
bool conv1x1_supported(int dtype, int K, int N, int epi);
int64_t conv1x1_partial_rows(int64_t m);      // upper bound of the statistics partial rows it writes
hipError_t launch_conv1x1(const RowsParams &p, hipStream_t s, int64_t *rows);   // *rows: partial rows written

// ---- persistent 3x3 CONV (weights and an input-row ring buffer in LDS) ----
bool conv3x3_supported(int dtype, int K, int N, int H, int W);
int64_t conv3x3_partial_rows(int64_t m);      // statistics partial rows it writes
hipError_t launch_conv3x3(const RowsParams &p, hipStream_t s);

// ---- weight gradient -------------------------------------------------------
enum { GB_DENSE = 0, GB_BNGRAD = 1, GB_POOLUP = 2 };
struct WgradParams {
    int dtype, k, n, h, w;
    int64_t m;
    int c_in, c_out;
    const void *x;                // conv input view
    int64_t x_ldc;
    int a_mode;                   // 0: x as is, 1: relu(bn(x)) recomputed on load, 2: relu(x)
    const float *a_gamma, *a_beta, *a_mean, *a_rstd;
    const float *a_ctr;           // a_mode 1: float32 centre of x (NULL: 0; a_mean relative to it)
    int gsrc;                     // GB_*
    const void *g;                // DENSE: [m][c_out] view; POOLUP: pooled gradient; BNGRAD: dy (dense)
    int64_t g_ldc;
    const void *gx;               // BNGRAD: BN input x view
    int64_t gx_ldc;
    const float *g_gamma, *g_mean, *g_rstd, *g_dgamma, *g_dbeta;
    int g_split;                  // GB_BNGRAD: 1 = summed gradient of several BNs (deferred_coef)
    const float *g_alpha, *g_betap;
    const float *g_ctr;           // GB_BNGRAD: float32 centre of gx (NULL: 0; g_mean relative to it)
    float *dw;                    // [k][k][c_in][c_out]
    float *part;                  // workspace for split partial tiles
    void *red;                    // split-K sum scratch (sum_partials_red_bytes)
};
size_t wgrad_ws_bytes(int dtype, int64_t m, int n, int h, int w, int c_in, int c_out, int k);
// *splits_out != NULL: launch the weight-gradient kernel only and report its
// split count (1: dw written directly; > 1: partial tiles in p.part for the
// caller to sum); NULL: the split-K sum is launched here as well.
hipError_t launch_wgrad(const WgradParams &p, hipStream_t s, int64_t *splits_out = nullptr);

// ---- network ends: first CONV, max pooling, classifier head (net_ends.hip) ----
// First CONV: 7x7, stride 2, pad 3, 64 output channels; the image is
// [n][h][w][kStemPix] with c_in <= kStemPix channels used per pixel.
constexpr int kStemK = 7, kStemPad = 3, kStemCout = 64, kStemPix = 4;
constexpr int kStemMaxW = 256;            // widest image
constexpr int kStemRows = 2;              // output rows per work item
constexpr int64_t kStemMaxGroups = 512;   // persistent workgroups (two per CU)
inline int stem_out(int x) { return (x + 2 * kStemPad - kStemK) / 2 + 1; }
struct StemParams {
    int n, h, w, ho, wo, c_in;
    const void *img;              // [n][h][w][kStemPix]
    const void *wt;               // [7][7][c_in][64]
    void *s;                      // forward output [n][ho][wo][64]
    float *part;                  // forward statistics partials [groups][2][64]
    const float *shift;           // forward statistics: sums of (s - shift) (NULL: 0)
    const void *g;                // weight gradient: DENSE g view / BNGRAD dy ([m][64] dense)
    int64_t g_ldc;
    const void *gx;               // BNGRAD: the BN input (the CONV output) view
    int64_t gx_ldc;
    const float *g_gamma, *g_mean, *g_rstd, *g_dgamma, *g_dbeta;
    const float *g_ctr;           // BNGRAD, float32: centre of gx (NULL: 0; g_mean relative to it)
    float *dwpart;                // weight-gradient partials [splits][7][7][c_in][64]
};
int64_t stem_groups(int64_t items);
int64_t stem_wgrad_splits(int dtype, int64_t items);
hipError_t launch_stem_conv(int dtype, const StemParams &p, bool stats, hipStream_t s);
hipError_t launch_stem_wgrad(int dtype, const StemParams &p, int gsrc, hipStream_t s);

// 3x3 / stride 2 / pad 1 max pooling (optionally of relu(bn(x))).
constexpr int kMaxPoolMaxC = 64;          // backward: channels
constexpr int kMaxPoolMaxWo = 64;         // backward: output width
constexpr int64_t kMaxPoolBwdGroups = 2048;
struct MaxPoolParams {
    int n, h, w, c, ho, wo;
    const void *x;                // input view [n][h][w][c]
    int64_t x_ldc;
    const float *gamma, *beta, *mean, *rstd;   // BN of x (NULL: plain pooling)
    const float *ctr;             // float32 centre of x (NULL: 0; mean relative to it)
    void *y;                      // forward: output view; backward: dy / dz (dense [n*h*w][c])
    int64_t y_ldc;
    const void *g;                // backward: gradient of the pooled output (view)
    int64_t g_ldc;
    float *part;                  // statistics / BN-backward partials [rows][2][c]
    const float *shift;           // forward statistics: sums of (y - shift) (NULL: 0)
};
int64_t maxpool_fwd_rows(int dtype, int64_t m_out, int c);
int64_t maxpool_bwd_groups(int n, int h);
hipError_t launch_maxpool_fwd(int dtype, const MaxPoolParams &p, bool bn, bool stats, hipStream_t s);
hipError_t launch_maxpool_bwd(int dtype, const MaxPoolParams &p, bool bn, hipStream_t s);

// Classifier head: BN -> ReLU -> global average pooling -> FC -> softmax CE.
enum { HB_SPLIT = 0, HB_SUMS = 1, HB_DX = 2 };
struct HeadParams {
    int n, h, w, c, classes;
    const void *x;                // [n*h*w][c] view
    int64_t x_ldc;
    const float *gamma, *beta, *mean, *rstd;
    const float *ctr;             // float32 centre of x (NULL: 0; mean relative to it)
    float *f;                     // pooled features [n][c]
    const void *wfc;              // [c][classes] (dtype)
    const float *bfc;             // [classes]
    const int32_t *labels;        // [n]
    float *logits, *dlogits, *loss;
    float *df, *dwfc, *dbfc;      // backward
    void *gx;                     // backward: summed term / input gradient view
    int64_t gx_ldc;
    const float *dgamma, *dbeta;  // HB_DX
    float *part;                  // BN-backward partials
};
int64_t head_rows(int dtype, int64_t m, int c);
hipError_t launch_head_fwd(int dtype, const HeadParams &p, hipStream_t s);
hipError_t launch_head_bwd_fc(int dtype, const HeadParams &p, hipStream_t s);
hipError_t launch_head_bn_bwd(int dtype, const HeadParams &p, int mode, hipStream_t s);

}  // namespace bnr
