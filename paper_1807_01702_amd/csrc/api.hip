// api.hip -- the C ABI of libbnr (declared in include/bnr.h): argument
// validation, workspace carving and the launch sequences of the fused
// BN fission/fusion path and of the unfused reference path.
//
// Every entry point validates all of its arguments before the first launch:
// on any error it returns without launching anything.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdarg>
#include <cstdio>
#include <cstring>

#include "../../include/bnr.h"
#include "kernels.hpp"
#include "tiles.hpp"
#include "trace.hpp"

using namespace bnr;

namespace {

thread_local char g_err[512] = "";

bnr_status fail(bnr_status s, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return s;
}

bnr_status ok()
{
    g_err[0] = 0;
    return BNR_OK;
}

bnr_status hip_status(hipError_t e, const char *what)
{
    if (e == hipSuccess) return BNR_OK;
    return fail(BNR_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

#define TRY(expr)                                        \
    do {                                                 \
        bnr_status _s = (expr);                          \
        if (_s != BNR_OK) return _s;                     \
    } while (0)
#define TRY_HIP(expr, what) TRY(hip_status((expr), what))

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }
inline int esize(bnr_dtype d) { return d == BNR_BF16 ? 2 : 4; }
inline int vec_of(bnr_dtype d) { return d == BNR_BF16 ? 8 : 4; }

bnr_status check_dtype(bnr_dtype d)
{
    if (d != BNR_F32 && d != BNR_BF16) return fail(BNR_ERR_DTYPE, "unknown dtype %d", (int)d);
    return BNR_OK;
}

bnr_status check_ptr(const void *p, const char *name, bool required = true)
{
    if (!p) return required ? fail(BNR_ERR_NULL, "%s is NULL", name) : BNR_OK;
    if (reinterpret_cast<uintptr_t>(p) % 16) return fail(BNR_ERR_ALIGN, "%s is not 16-byte aligned", name);
    return BNR_OK;
}

bnr_status check_fptr(const float *p, const char *name)
{
    if (!p) return fail(BNR_ERR_NULL, "%s is NULL", name);
    if (reinterpret_cast<uintptr_t>(p) % 4) return fail(BNR_ERR_ALIGN, "%s is not 4-byte aligned", name);
    return BNR_OK;
}

bnr_status check_channels(int c, int ldc, bnr_dtype d, const char *what)
{
    if (c <= 0 || ldc <= 0) return fail(BNR_ERR_SHAPE, "%s: channels %d / ldc %d must be positive", what, c, ldc);
    if (ldc < c) return fail(BNR_ERR_SHAPE, "%s: ldc %d < channels %d", what, ldc, c);
    if (c % vec_of(d) || ldc % vec_of(d))
        return fail(BNR_ERR_ALIGN, "%s: channels %d and ldc %d must be multiples of %d", what, c, ldc, vec_of(d));
    return BNR_OK;
}

// byte range [lo, hi) of a pixel-strided view
struct Range { uintptr_t lo, hi; };
Range view_range(const void *p, int64_t m, int64_t c, int64_t ldc, int es)
{
    uintptr_t lo = reinterpret_cast<uintptr_t>(p);
    return Range{lo, lo + (uintptr_t)(((m - 1) * ldc + c) * es)};
}
bool overlap(Range a, Range b) { return a.lo < b.hi && b.lo < a.hi; }

bnr_status check_bn(const bnr_bn *bn, const char *name, bool need_affine, bool need_stats_out)
{
    if (!bn) return fail(BNR_ERR_NULL, "%s is NULL", name);
    if (need_affine) {
        TRY(check_fptr(bn->gamma, "bn.gamma"));
        TRY(check_fptr(bn->beta, "bn.beta"));
    }
    TRY(check_fptr(bn->mean, "bn.mean"));
    TRY(check_fptr(bn->rstd, "bn.rstd"));
    if (bn->var && reinterpret_cast<uintptr_t>(bn->var) % 4) return fail(BNR_ERR_ALIGN, "bn.var misaligned");
    if (need_stats_out && !(bn->eps > 0.0f)) return fail(BNR_ERR_SHAPE, "%s.eps must be > 0", name);
    if (need_stats_out) {
        const auto mis = [](const void *q) { return reinterpret_cast<uintptr_t>(q) % 4 != 0; };
        if (mis(bn->shift) || mis(bn->running_mean) || mis(bn->running_var) || mis(bn->mean_lo))
            return fail(BNR_ERR_ALIGN, "%s shift / running statistics / mean_lo misaligned", name);
        const float *mr = bn->mean_lo;
        if (mr && (mr == bn->mean || mr == bn->shift || mr == bn->var || mr == bn->rstd || mr == bn->running_mean ||
                   mr == bn->running_var))
            return fail(BNR_ERR_ALIAS, "%s.mean_lo aliases another array of the BN", name);
        if (bn->running_var && !bn->running_mean)
            return fail(BNR_ERR_NULL, "%s.running_var set without running_mean", name);
        if (bn->running_mean && !(bn->momentum >= 0.0f && bn->momentum <= 1.0f))
            return fail(BNR_ERR_SHAPE, "%s.momentum must be in [0, 1]", name);
    }
    return BNR_OK;
}

// forward finalisation terms of a statistics producer: the one-sweep shift
// (FIN_MVF) and the running statistics
SplitTerms fwd_terms(const bnr_bn *bn, bool one_sweep)
{
    SplitTerms t{nullptr, nullptr, nullptr, nullptr, 0, one_sweep ? bn->shift : nullptr, bn->running_mean,
                 bn->running_var, bn->momentum, one_sweep ? bn->mean_lo : nullptr};
    return t;
}

// terms of a two-pass mean combine (FIN_MEAN): the low part of the mean
SplitTerms mean_terms(const bnr_bn *bn)
{
    SplitTerms t{nullptr, nullptr, nullptr, nullptr, 0, nullptr, nullptr, nullptr, 0.f, bn->mean_lo};
    return t;
}

// The mean a consumer of bn's input is given and the centre it subtracts from
// the input first (bn_centre): float32 data with mean_lo set is normalised as
// (x - mean) - mean_lo, everything else as x - mean.
struct Centred { const float *mean, *ctr; };
Centred centred(const bnr_bn *bn, int dtype)
{
    if (dtype == DT_F32 && bn->mean_lo) return Centred{bn->mean_lo, bn->mean};
    return Centred{bn->mean, nullptr};
}

bnr_status check_desc(const bnr_conv_desc *d)
{
    if (!d) return fail(BNR_ERR_NULL, "desc is NULL");
    TRY(check_dtype(d->dtype));
    if (d->n <= 0 || d->h <= 0 || d->w <= 0) return fail(BNR_ERR_SHAPE, "n, h, w must be positive");
    if (d->k != 1 && d->k != 3) return fail(BNR_ERR_UNSUPPORTED, "filter size %d (only 1 and 3)", d->k);
    if (d->k == 3 && d->w > kRowsMaxW3)
        return fail(BNR_ERR_UNSUPPORTED, "3x3 CONV with image width %d > %d", d->w, kRowsMaxW3);
    const int64_t m = (int64_t)d->n * d->h * d->w;
    if (m > (int64_t)1 << 31) return fail(BNR_ERR_SHAPE, "too many pixels (%lld)", (long long)m);
    TRY(check_channels(d->c_in, d->in_ldc, d->dtype, "conv input"));
    TRY(check_channels(d->c_out, d->out_ldc, d->dtype, "conv output"));
    if (d->c_in > 2048 || d->c_out > 2048) return fail(BNR_ERR_UNSUPPORTED, "more than 2048 channels");
    return BNR_OK;
}

int64_t pixels(const bnr_conv_desc *d) { return (int64_t)d->n * d->h * d->w; }

// workspace regions for the conv entry points:
//   pack  | packed weights (forward or data-gradient layout)
//   part  | per-tile statistics partial sums [tiles][2][C]
//   red   | statistics combine scratch (float64 level 1)
//   wg    | weight-gradient split partial tiles
//   wgred | split-K sum scratch
struct ConvWs { size_t pack, part, red, wg, wgred, total; };
ConvWs conv_ws(const bnr_conv_desc *d)
{
    const int taps = d->k * d->k, dt = d->dtype == BNR_BF16 ? DT_BF16 : DT_F32;
    const int64_t m = pixels(d);
    ConvWs w;
    size_t pf = rows_pack_bytes(dt, taps, d->c_in, d->c_out), pb = rows_pack_bytes(dt, taps, d->c_out, d->c_in);
    w.pack = align_up(pf > pb ? pf : pb);
    size_t sf = (size_t)rows_mtiles(dt, taps, m, d->c_out) * 2 * d->c_out * 4;
    size_t sb = (size_t)rows_mtiles(dt, taps, m, d->c_in) * 2 * d->c_in * 4;
    size_t ss = (size_t)stats_row_blocks(m, d->c_in, dt) * 2 * d->c_in * 4;
    const int cmax = d->c_in > d->c_out ? d->c_in : d->c_out;
    const int64_t prow = conv1x1_partial_rows(m) > conv3x3_partial_rows(m) ? conv1x1_partial_rows(m)
                                                                            : conv3x3_partial_rows(m);
    const size_t sp = (size_t)prow * 2 * cmax * 4;
    size_t part = sf > sb ? sf : sb;
    if (sp > part) part = sp;
    w.part = align_up(part > ss ? part : ss);
    w.red = align_up(stats_red_bytes(d->c_in > d->c_out ? d->c_in : d->c_out));
    w.wg = align_up(wgrad_ws_bytes(dt, m, d->n, d->h, d->w, d->c_in, d->c_out, d->k));
    w.wgred = align_up(sum_partials_red_bytes((int64_t)d->k * d->k * d->c_in * d->c_out));
    w.total = w.pack + w.part + w.red + w.wg + w.wgred;
    return w;
}

struct ConvPtrs { void *pack; float *part; void *red; float *wg; void *wgred; };
ConvPtrs conv_ptrs(void *ws, const ConvWs &w)
{
    char *b = (char *)ws;
    return ConvPtrs{b, (float *)(b + w.pack), b + w.pack + w.part, (float *)(b + w.pack + w.part + w.red),
                    b + w.pack + w.part + w.red + w.wg};
}

size_t stats_part_bytes(int64_t m, int c)
{
    size_t a = (size_t)stats_row_blocks(m, c, DT_BF16) * 2 * c * 4;
    size_t b = (size_t)stats_row_blocks(m, c, DT_F32) * 2 * c * 4;
    return align_up(a > b ? a : b);
}

size_t stats_ws(int64_t m, int c) { return stats_part_bytes(m, c) + align_up(stats_red_bytes(c)); }

bnr_status check_ws(void *ws, size_t have, size_t need)
{
    if (need == 0) return BNR_OK;
    if (!ws) return fail(BNR_ERR_WORKSPACE, "workspace is NULL (%zu bytes needed)", need);
    if (reinterpret_cast<uintptr_t>(ws) % kAlign) return fail(BNR_ERR_ALIGN, "workspace not 256-byte aligned");
    if (have < need) return fail(BNR_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", have, need);
    return BNR_OK;
}

int dt_of(bnr_dtype d) { return d == BNR_BF16 ? DT_BF16 : DT_F32; }

// statistics of a [m][c] view: partial sweep + float64 combine (MVF)
bnr_status run_stats(int64_t m, int c, int ldc, bnr_dtype dt, const void *x, bnr_bn *bn, void *ws, hipStream_t s)
{
    const int64_t R = stats_row_blocks(m, c, dt_of(dt));
    float *part = (float *)ws;
    void *red = (char *)ws + stats_part_bytes(m, c);
    TRY_HIP(launch_stats_partial(dt_of(dt), x, ldc, m, c, ST_SUMSQ, bn->shift, nullptr, nullptr, 0, part, R, s),
            "stats sweep");
    const SplitTerms ft = fwd_terms(bn, true);
    TRY_HIP(launch_stats_finalize(part, R, c, m, FIN_MVF, bn->eps, bn->mean, bn->var, bn->rstd, nullptr, nullptr, red,
                                  s, &ft),
            "stats combine");
    return BNR_OK;
}

bnr_status validate_grad_src(const bnr_conv_desc *d, const bnr_grad_src *g)
{
    if (!g) return fail(BNR_ERR_NULL, "g_src is NULL");
    const int es = esize(d->dtype);
    const int64_t m = pixels(d);
    if (g->kind == BNR_GRAD_DENSE) {
        TRY(check_ptr(g->g, "g_src.g"));
        TRY(check_channels(d->c_out, g->g_ldc, d->dtype, "g_src.g"));
        (void)view_range(g->g, m, d->c_out, g->g_ldc, es);
    } else if (g->kind == BNR_GRAD_BN) {
        TRY(check_ptr(g->dy, "g_src.dy"));
        TRY(check_ptr(g->x, "g_src.x"));
        TRY(check_channels(d->c_out, g->x_ldc, d->dtype, "g_src.x"));
        TRY(check_bn(g->bn, "g_src.bn", true, false));
        TRY(check_fptr(g->dgamma, "g_src.dgamma"));
        TRY(check_fptr(g->dbeta, "g_src.dbeta"));
    } else if (g->kind == BNR_GRAD_AVGPOOL2) {
        TRY(check_ptr(g->g, "g_src.g"));
        TRY(check_channels(d->c_out, g->g_ldc, d->dtype, "g_src.g (pooled)"));
        if (d->h % 2 || d->w % 2) return fail(BNR_ERR_SHAPE, "average-pooling gradient needs even h, w");
    } else if (g->kind == BNR_GRAD_SPLIT) {
        TRY(check_ptr(g->g, "g_src.g"));
        TRY(check_channels(d->c_out, g->g_ldc, d->dtype, "g_src.g (summed)"));
        TRY(check_ptr(g->x, "g_src.x"));
        TRY(check_channels(d->c_out, g->x_ldc, d->dtype, "g_src.x"));
        TRY(check_bn(g->bn, "g_src.bn", false, false));
        TRY(check_fptr(g->alpha, "g_src.alpha"));
        TRY(check_fptr(g->betap, "g_src.betap"));
    } else {
        return fail(BNR_ERR_UNSUPPORTED, "unknown gradient kind %d", (int)g->kind);
    }
    return BNR_OK;
}

void fill_rows(RowsParams &rp, const bnr_conv_desc *d, int K, int N)
{
    memset(&rp, 0, sizeof rp);
    rp.dtype = dt_of(d->dtype);
    rp.taps = d->k * d->k;
    rp.n = d->n; rp.h = d->h; rp.w = d->w;
    rp.m = pixels(d);
    rp.K = K; rp.N = N;
}

// Runs the CONV GEMM of rp (forward when transpose = 0, data gradient when 1)
// with the persistent 1x1 kernel when it applies, else packs the weights and
// runs the tiled kernel.  *rows = statistics partial rows written.
bnr_status launch_conv_any(RowsParams &rp, const bnr_conv_desc *d, const void *w, int transpose, void *wpack,
                           int64_t *rows, hipStream_t s)
{
    if (rp.taps == 1 && conv1x1_supported(rp.dtype, rp.K, rp.N, rp.epi)) {
        rp.wraw = w;
        rp.wtrans = transpose;
        TRY_HIP(launch_conv1x1(rp, s, rows), transpose ? "conv data gradient" : "conv forward");
        return BNR_OK;
    }
    if (rp.taps == 9 && rp.pro != PRO_POOLUP && !rp.e_scale && conv3x3_supported(rp.dtype, rp.K, rp.N, rp.h, rp.w)) {
        rp.wraw = w;
        rp.wtrans = transpose;
        *rows = conv3x3_partial_rows(rp.m);
        TRY_HIP(launch_conv3x3(rp, s), transpose ? "conv data gradient" : "conv forward");
        return BNR_OK;
    }
    if (rows_direct_weights(rp.dtype, rp.taps, rp.m, rp.K, rp.N, rp.a_ldc, rp.a2_ldc, rp.pro, rp.side != nullptr)) {
        rp.wdirect = 1;                 // bf16 1x1: the tiled kernel reads the caller's weights, no packing
        rp.wraw = w;
        rp.wtrans = transpose;
    } else {
        TRY_HIP(launch_pack_weights(rp.dtype, w, d->k, d->c_in, d->c_out, transpose, wpack, s), "weight packing");
        rp.wpack = wpack;
    }
    *rows = rows_mtiles(rp.dtype, rp.taps, rp.m, rp.N);
    TRY_HIP(launch_conv_rows(rp, s), transpose ? "conv data gradient" : "conv forward");
    return BNR_OK;
}

// workspace bytes a forward CONV touches: the first three regions (packed
// weights, statistics partial rows, combine stage)
size_t conv_fwd_ws(const ConvWs &w) { return w.pack + w.part + w.red; }

// forward CONV with optional BN+ReLU prologue and optional statistics epilogue
// (need: the workspace bytes checked; 0 = the whole conv workspace).  pool:
// the BN+ReLU output is averaged over 2x2 windows before the 1x1 CONV, whose
// output y is the pooled [n][h/2][w/2][c_out] view.  z (BN+ReLU forward,
// not pooled): the BN+ReLU output is also written to the view z (pixel stride
// z_ldc), the materialised O2' sweep.
bnr_status conv_fwd(const bnr_conv_desc *d, const void *x, const bnr_bn *x_bn, const void *w, void *y,
                    bnr_bn *y_bn, void *ws, size_t ws_bytes, void *stream, size_t need = 0, bool pool = false,
                    void *z = nullptr, int32_t z_ldc = 0)
{
    TRY(check_desc(d));
    if (z && (pool || !x_bn)) return fail(BNR_ERR_UNSUPPORTED, "z is written by the BN+ReLU forward only");
    if (pool && (d->k != 1 || d->h % 2 || d->w % 2 || !x_bn))
        return fail(d->k != 1 ? BNR_ERR_UNSUPPORTED : BNR_ERR_SHAPE,
                    "pooled forward: 1x1 CONV with BN, even h and w (k %d, h %d, w %d)", d->k, d->h, d->w);
    TRY(check_ptr(x, "x"));
    TRY(check_ptr(w, "w"));
    TRY(check_ptr(y, "y"));
    if (x_bn) TRY(check_bn(x_bn, "x_bn", true, false));
    if (y_bn) TRY(check_bn(y_bn, "y_bn", false, true));
    const ConvWs cw = conv_ws(d);
    TRY(check_ws(ws, ws_bytes, need ? need : cw.total));
    const int es = esize(d->dtype);
    const int64_t m = pixels(d);
    const int64_t my = pool ? m / 4 : m;                 // output rows
    Range ry = view_range(y, my, d->c_out, d->out_ldc, es);
    if (overlap(ry, view_range(x, m, d->c_in, d->in_ldc, es))) return fail(BNR_ERR_ALIAS, "y overlaps x");
    const int64_t wbytes = (int64_t)d->k * d->k * d->c_in * d->c_out * es;
    Range rw{reinterpret_cast<uintptr_t>(w), reinterpret_cast<uintptr_t>(w) + (uintptr_t)wbytes};
    if (overlap(ry, rw)) return fail(BNR_ERR_ALIAS, "y overlaps w");
    if (z) {
        TRY(check_channels(d->c_in, z_ldc, d->dtype, "z"));
        const Range rz = view_range(z, m, d->c_in, z_ldc, es);
        if (overlap(rz, view_range(x, m, d->c_in, d->in_ldc, es)) || overlap(rz, ry) || overlap(rz, rw))
            return fail(BNR_ERR_ALIAS, "z overlaps x, y or w");
    }

    hipStream_t s = (hipStream_t)stream;
    const ConvPtrs wp = conv_ptrs(ws, cw);
    void *wpack = wp.pack;
    float *part = wp.part;
    RowsParams rp;
    fill_rows(rp, d, d->c_in, d->c_out);
    rp.pro = x_bn ? (pool ? PRO_BNRELU_POOL : PRO_BNRELU) : PRO_NONE;
    rp.m = my;
    rp.a = x; rp.a_ldc = d->in_ldc;
    if (x_bn) {
        const Centred cx = centred(x_bn, rp.dtype);
        rp.p_gamma = x_bn->gamma; rp.p_beta = x_bn->beta; rp.p_mean = cx.mean; rp.p_rstd = x_bn->rstd;
        rp.p_ctr = cx.ctr;
    }
    rp.side = z; rp.side_ldc = z_ldc;
    rp.epi = y_bn ? EPI_STATS : EPI_STORE;
    rp.y = y; rp.y_ldc = d->out_ldc;
    rp.part = part;
    rp.e_shift = y_bn ? y_bn->shift : nullptr;
    int64_t R = 0;
    TRY(launch_conv_any(rp, d, w, 0, wpack, &R, s));
    if (y_bn) {
        const SplitTerms ft = fwd_terms(y_bn, true);
        TRY_HIP(launch_stats_finalize(part, R, d->c_out, my, FIN_MVF, y_bn->eps, y_bn->mean, y_bn->var, y_bn->rstd,
                                      nullptr, nullptr, wp.red, s, &ft),
                "stats combine");
    }
    return ok();
}

}  // namespace

// ---- scratch of the entry point that allocates nothing ----
// bnr_bn_relu_conv_fwd_static keeps its forward workspace (packed weights,
// statistics partial rows, the combine's float64 stage) in this array: one
// copy per GPU, alive until the process ends.  Host code never uses the
// array's name as an address (on the host it is a stand-in symbol, not
// device memory): the device address comes from hipGetSymbolAddress, taken
// once per device with that device current.
constexpr size_t kStaticScratchBytes = (size_t)16 << 20;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::atomic<void *> g_scratch_ptr[kMaxDevices];

// device address of `scratch` on the current device (looked up on the first
// call on that device; concurrent first calls look up the same address)
bnr_status static_scratch(void **out)
{
    int dev = -1;
    TRY_HIP(hipGetDevice(&dev), "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices) return fail(BNR_ERR_UNSUPPORTED, "device ordinal %d >= %d", dev, kMaxDevices);
    void *p = g_scratch_ptr[dev].load(std::memory_order_acquire);
    if (!p) {
        TRY_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)");
        if (!p) return fail(BNR_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
        if (reinterpret_cast<uintptr_t>(p) % kAlign) return fail(BNR_ERR_HIP, "scratch is not 256-byte aligned");
        g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
    *out = p;
    return BNR_OK;
}

}  // namespace

extern "C" {

const char *bnr_status_string(bnr_status s)
{
    switch (s) {
    case BNR_OK: return "BNR_OK";
    case BNR_ERR_NULL: return "BNR_ERR_NULL";
    case BNR_ERR_SHAPE: return "BNR_ERR_SHAPE";
    case BNR_ERR_DTYPE: return "BNR_ERR_DTYPE";
    case BNR_ERR_ALIGN: return "BNR_ERR_ALIGN";
    case BNR_ERR_WORKSPACE: return "BNR_ERR_WORKSPACE";
    case BNR_ERR_UNSUPPORTED: return "BNR_ERR_UNSUPPORTED";
    case BNR_ERR_HIP: return "BNR_ERR_HIP";
    case BNR_ERR_ALIAS: return "BNR_ERR_ALIAS";
    }
    return "BNR_ERR_UNKNOWN";
}

const char *bnr_last_error(void) { return g_err; }

size_t bnr_stats_workspace_size(int64_t m, int32_t c)
{
    if (m <= 0 || c <= 0) return 0;
    return stats_ws(m, c);
}

size_t bnr_workspace_size(const bnr_conv_desc *d)
{
    if (check_desc(d) != BNR_OK) return 0;
    return conv_ws(d).total;
}

bnr_status bnr_bn_stats(int64_t m, int32_t c, int32_t ldc, bnr_dtype dtype, const void *x, bnr_bn *bn, void *ws,
                        size_t ws_bytes, void *stream)
{
    TRY(check_dtype(dtype));
    if (m <= 0 || m > ((int64_t)1 << 31)) return fail(BNR_ERR_SHAPE, "m = %lld out of range", (long long)m);
    TRY(check_channels(c, ldc, dtype, "x"));
    TRY(check_ptr(x, "x"));
    TRY(check_bn(bn, "bn", false, true));
    TRY(check_ws(ws, ws_bytes, stats_ws(m, c)));
    TRY(run_stats(m, c, ldc, dtype, x, bn, ws, (hipStream_t)stream));
    return ok();
}

bnr_status bnr_conv_bn_stats_fwd(const bnr_conv_desc *d, const void *x, const void *w, void *y, bnr_bn *y_bn,
                                 void *ws, size_t ws_bytes, void *stream)
{
    if (!y_bn) return fail(BNR_ERR_NULL, "y_bn is NULL");
    return conv_fwd(d, x, nullptr, w, y, y_bn, ws, ws_bytes, stream);
}

bnr_status bnr_bn_relu_conv_fwd(const bnr_conv_desc *d, const void *x, const bnr_bn *x_bn, const void *w, void *y,
                                bnr_bn *y_bn, void *ws, size_t ws_bytes, void *stream)
{
    if (!x_bn) return fail(BNR_ERR_NULL, "x_bn is NULL");
    return conv_fwd(d, x, x_bn, w, y, y_bn, ws, ws_bytes, stream);
}

bnr_status bnr_bn_relu_conv_fwd_o2(const bnr_conv_desc *d, const void *x, const bnr_bn *x_bn, const void *w,
                                   void *y, bnr_bn *y_bn, void *z, int32_t z_ldc, void *ws, size_t ws_bytes,
                                   void *stream)
{
    if (!x_bn) return fail(BNR_ERR_NULL, "x_bn is NULL");
    if (!z) return fail(BNR_ERR_NULL, "z is NULL");
    return conv_fwd(d, x, x_bn, w, y, y_bn, ws, ws_bytes, stream, 0, false, z, z_ldc);
}

bnr_status bnr_bn_relu_conv_fwd_static(const bnr_conv_desc *d, const void *x, const bnr_bn *x_bn, const void *w,
                                       void *y, bnr_bn *y_bn, void *stream)
{
    if (!x_bn) return fail(BNR_ERR_NULL, "x_bn is NULL");
    TRY(check_desc(d));
    const size_t need = conv_fwd_ws(conv_ws(d));
    if (need > kStaticScratchBytes)
        return fail(BNR_ERR_WORKSPACE, "this CONV needs %zu bytes of scratch, more than the %zu of the static array",
                    need, kStaticScratchBytes);
    void *ptr = nullptr;
    TRY(static_scratch(&ptr));
    TraceSuppress no_events;              // launch timing would create HIP events
    return conv_fwd(d, x, x_bn, w, y, y_bn, ptr, kStaticScratchBytes, stream, need);
}

bnr_status bnr_bn_add_relu_conv_fwd(const bnr_conv_desc *d, const void *y, const bnr_bn *y_bn, const void *ident,
                                    int32_t ident_ldc, void *r, int32_t r_ldc, const void *w, void *out,
                                    bnr_bn *out_bn, void *ws, size_t ws_bytes, void *stream)
{
    TRY(check_desc(d));
    if (d->k != 1) return fail(BNR_ERR_UNSUPPORTED, "residual prologue: 1x1 CONV only (k = %d)", d->k);
    TRY(check_ptr(y, "y"));
    TRY(check_ptr(ident, "ident"));
    TRY(check_ptr(r, "r"));
    TRY(check_ptr(w, "w"));
    TRY(check_ptr(out, "out"));
    TRY(check_channels(d->c_in, ident_ldc, d->dtype, "ident"));
    TRY(check_channels(d->c_in, r_ldc, d->dtype, "r"));
    TRY(check_bn(y_bn, "y_bn", true, false));
    if (out_bn) TRY(check_bn(out_bn, "out_bn", false, true));
    const ConvWs cw = conv_ws(d);
    TRY(check_ws(ws, ws_bytes, cw.total));
    const int es = esize(d->dtype);
    const int64_t m = pixels(d);
    const Range ry = view_range(y, m, d->c_in, d->in_ldc, es), ri = view_range(ident, m, d->c_in, ident_ldc, es);
    const Range rr = view_range(r, m, d->c_in, r_ldc, es), ro = view_range(out, m, d->c_out, d->out_ldc, es);
    const int64_t wbytes = (int64_t)d->c_in * d->c_out * es;
    const Range rw{reinterpret_cast<uintptr_t>(w), reinterpret_cast<uintptr_t>(w) + (uintptr_t)wbytes};
    if (overlap(rr, ry) || overlap(rr, ri) || overlap(rr, rw) || overlap(rr, ro))
        return fail(BNR_ERR_ALIAS, "r overlaps y, ident, w or out");
    if (overlap(ro, ry) || overlap(ro, ri) || overlap(ro, rw)) return fail(BNR_ERR_ALIAS, "out overlaps y, ident or w");

    hipStream_t s = (hipStream_t)stream;
    const ConvPtrs wp = conv_ptrs(ws, cw);
    RowsParams rp;
    fill_rows(rp, d, d->c_in, d->c_out);
    rp.pro = PRO_BNADDRELU;
    rp.a = y; rp.a_ldc = d->in_ldc;
    rp.a2 = ident; rp.a2_ldc = ident_ldc;
    const Centred cy = centred(y_bn, rp.dtype);
    rp.p_gamma = y_bn->gamma; rp.p_beta = y_bn->beta; rp.p_mean = cy.mean; rp.p_rstd = y_bn->rstd;
    rp.p_ctr = cy.ctr;
    rp.side = r; rp.side_ldc = r_ldc;
    rp.epi = out_bn ? EPI_STATS : EPI_STORE;
    rp.y = out; rp.y_ldc = d->out_ldc;
    rp.part = wp.part;
    rp.e_shift = out_bn ? out_bn->shift : nullptr;
    int64_t R = 0;
    TRY(launch_conv_any(rp, d, w, 0, wp.pack, &R, s));
    if (out_bn) {
        const SplitTerms ft = fwd_terms(out_bn, true);
        TRY_HIP(launch_stats_finalize(wp.part, R, d->c_out, m, FIN_MVF, out_bn->eps, out_bn->mean, out_bn->var,
                                      out_bn->rstd, nullptr, nullptr, wp.red, s, &ft),
                "stats combine");
    }
    return ok();
}

bnr_status bnr_bn_relu_conv_pool_fwd(const bnr_conv_desc *d, const void *x, const bnr_bn *x_bn, const void *w,
                                     void *y, bnr_bn *y_bn, void *ws, size_t ws_bytes, void *stream)
{
    if (!x_bn) return fail(BNR_ERR_NULL, "x_bn is NULL");
    return conv_fwd(d, x, x_bn, w, y, y_bn, ws, ws_bytes, stream, 0, true);
}

bnr_status bnr_avgpool2_fwd(int32_t n, int32_t h, int32_t w, int32_t c, bnr_dtype dtype, const void *x, int32_t ldc,
                            void *y, int32_t y_ldc, void *stream)
{
    TRY(check_dtype(dtype));
    if (n <= 0 || h <= 0 || w <= 0) return fail(BNR_ERR_SHAPE, "n, h, w must be positive");
    if (h % 2 || w % 2) return fail(BNR_ERR_SHAPE, "h and w must be even");
    TRY(check_channels(c, ldc, dtype, "x"));
    TRY(check_channels(c, y_ldc, dtype, "y"));
    TRY(check_ptr(x, "x"));
    TRY(check_ptr(y, "y"));
    const int es = esize(dtype);
    const int64_t m = (int64_t)n * h * w;
    if (overlap(view_range(x, m, c, ldc, es), view_range(y, m / 4, c, y_ldc, es)))
        return fail(BNR_ERR_ALIAS, "y overlaps x");
    TRY_HIP(launch_avgpool2(dt_of(dtype), n, h, w, c, x, ldc, y, y_ldc, (hipStream_t)stream), "avgpool");
    return ok();
}

bnr_status bnr_avgpool2_bwd(int32_t n, int32_t h, int32_t w, int32_t c, bnr_dtype dtype, const void *g, int32_t g_ldc,
                            void *gx, int32_t gx_ldc, void *stream)
{
    TRY(check_dtype(dtype));
    if (n <= 0 || h <= 0 || w <= 0) return fail(BNR_ERR_SHAPE, "n, h, w must be positive");
    if (h % 2 || w % 2) return fail(BNR_ERR_SHAPE, "h and w must be even");
    TRY(check_channels(c, g_ldc, dtype, "g"));
    TRY(check_channels(c, gx_ldc, dtype, "gx"));
    TRY(check_ptr(g, "g"));
    TRY(check_ptr(gx, "gx"));
    const int es = esize(dtype);
    const int64_t m = (int64_t)n * h * w;
    if (overlap(view_range(gx, m, c, gx_ldc, es), view_range(g, m / 4, c, g_ldc, es)))
        return fail(BNR_ERR_ALIAS, "gx overlaps g");
    TRY_HIP(launch_avgpool2_bwd(dt_of(dtype), n, h, w, c, g, g_ldc, gx, gx_ldc, (hipStream_t)stream),
            "avgpool backward");
    return ok();
}

// Steps 1-3 of the fused backward on validated arguments: data gradient with
// the gradient-source prologue and (x_bn) the BN-backward epilogue into y
// (dy, or with y_scale the summed-gradient term gamma*rstd*dy, y_acc: added),
// the dbeta/dgamma combine (with split: also alpha/betap), the weight gradient.
enum { BWD_DATA = 1, BWD_WEIGHTS = 2 };

// z (with x_bn): the stored BN+ReLU output of the forward (O2'), read by the
// BN-backward epilogue in place of x and by the weight gradient as its operand.
static bnr_status bwd_steps(const bnr_conv_desc *d, const void *x, const bnr_bn *x_bn, const void *w,
                            const bnr_grad_src *g, float *dw, float *dgamma, float *dbeta, void *y, int64_t y_ldc,
                            int y_scale, int y_acc, const SplitTerms *split, void *ws, hipStream_t s,
                            int parts = BWD_DATA | BWD_WEIGHTS, const void *z = nullptr, int64_t z_ldc = 0)
{
    const ConvWs cw = conv_ws(d);
    const ConvPtrs cp = conv_ptrs(ws, cw);
    const int64_t m = pixels(d);
    const int dt = dt_of(d->dtype);

    // 1. data gradient.  With both halves in this call and few enough partial
    // rows, the dbeta/dgamma combine (step 2) rides in the launch that sums
    // the weight gradient's split-K partials (after step 3).
    int64_t R = 0;
    bool tail_combine = false;
    if (parts & BWD_DATA) {
    RowsParams rp;
    fill_rows(rp, d, d->c_out, d->c_in);
    if (g->kind == BNR_GRAD_DENSE) {
        rp.pro = PRO_NONE; rp.a = g->g; rp.a_ldc = g->g_ldc;
    } else if (g->kind == BNR_GRAD_BN) {
        rp.pro = PRO_BNGRAD; rp.a = g->dy; rp.a_ldc = d->c_out; rp.a2 = g->x; rp.a2_ldc = g->x_ldc;
        const Centred cg = centred(g->bn, rp.dtype);
        rp.p_gamma = g->bn->gamma; rp.p_mean = cg.mean; rp.p_rstd = g->bn->rstd; rp.p_ctr = cg.ctr;
        rp.p_dgamma = g->dgamma; rp.p_dbeta = g->dbeta;
    } else if (g->kind == BNR_GRAD_SPLIT) {
        rp.pro = PRO_BNGRAD; rp.p_split = 1; rp.a = g->g; rp.a_ldc = g->g_ldc; rp.a2 = g->x; rp.a2_ldc = g->x_ldc;
        const Centred cg = centred(g->bn, rp.dtype);
        rp.p_mean = cg.mean; rp.p_rstd = g->bn->rstd; rp.p_alpha = g->alpha; rp.p_betap = g->betap;
        rp.p_ctr = cg.ctr;
    } else {
        rp.pro = PRO_POOLUP; rp.a = g->g; rp.a_ldc = g->g_ldc;
    }
    if (x_bn) {
        rp.epi = EPI_BNBWD; rp.y = y; rp.y_ldc = y_ldc; rp.part = cp.part;
        rp.e_scale = y_scale; rp.accumulate = y_scale && y_acc ? 1 : 0;
        rp.ex = x; rp.ex_ldc = d->in_ldc;
        const Centred cx = centred(x_bn, rp.dtype);
        rp.e_gamma = x_bn->gamma; rp.e_beta = x_bn->beta; rp.e_mean = cx.mean; rp.e_rstd = x_bn->rstd;
        rp.e_ctr = cx.ctr;
        if (z) { rp.e_zsrc = 1; rp.ex = z; rp.ex_ldc = z_ldc; rp.ex2 = x; rp.ex2_ldc = d->in_ldc; }
    } else {
        rp.epi = EPI_STORE; rp.y = y; rp.y_ldc = y_ldc; rp.accumulate = y_acc ? 1 : 0;
    }
    TRY(launch_conv_any(rp, d, w, 1, cp.pack, &R, s));
    // 2. dbeta = sum(dy), dgamma = sum(dy * xhat)
    tail_combine = x_bn && (parts & BWD_WEIGHTS) && R <= kCombineOneMaxRows;
    if (x_bn && !tail_combine) {
        TRY_HIP(launch_stats_finalize(cp.part, R, d->c_in, m, FIN_BWD, 0.f, nullptr, nullptr, nullptr, dbeta, dgamma,
                                      cp.red, s, split),
                "backward sums combine");
    }
    }
    if (!(parts & BWD_WEIGHTS)) return BNR_OK;
    // 3. weight gradient, both operands recomputed on load (z: read as it is)
    WgradParams wp;
    memset(&wp, 0, sizeof wp);
    wp.dtype = dt; wp.k = d->k; wp.n = d->n; wp.h = d->h; wp.w = d->w; wp.m = m;
    wp.c_in = d->c_in; wp.c_out = d->c_out;
    wp.x = z ? z : x; wp.x_ldc = z ? z_ldc : d->in_ldc;
    if (x_bn && !z) {
        wp.a_mode = 1;
        const Centred cx = centred(x_bn, dt);
        wp.a_gamma = x_bn->gamma; wp.a_beta = x_bn->beta; wp.a_mean = cx.mean; wp.a_rstd = x_bn->rstd;
        wp.a_ctr = cx.ctr;
    }
    if (g->kind == BNR_GRAD_DENSE) {
        wp.gsrc = GB_DENSE; wp.g = g->g; wp.g_ldc = g->g_ldc;
    } else if (g->kind == BNR_GRAD_BN) {
        const Centred cg = centred(g->bn, dt);
        wp.gsrc = GB_BNGRAD; wp.g = g->dy; wp.g_ldc = d->c_out; wp.gx = g->x; wp.gx_ldc = g->x_ldc;
        wp.g_gamma = g->bn->gamma; wp.g_mean = cg.mean; wp.g_rstd = g->bn->rstd; wp.g_ctr = cg.ctr;
        wp.g_dgamma = g->dgamma; wp.g_dbeta = g->dbeta;
    } else if (g->kind == BNR_GRAD_SPLIT) {
        const Centred cg = centred(g->bn, dt);
        wp.gsrc = GB_BNGRAD; wp.g_split = 1; wp.g = g->g; wp.g_ldc = g->g_ldc; wp.gx = g->x; wp.gx_ldc = g->x_ldc;
        wp.g_mean = cg.mean; wp.g_rstd = g->bn->rstd; wp.g_alpha = g->alpha; wp.g_betap = g->betap;
        wp.g_ctr = cg.ctr;
    } else {
        wp.gsrc = GB_POOLUP; wp.g = g->g; wp.g_ldc = g->g_ldc;
    }
    wp.dw = dw; wp.part = cp.wg; wp.red = cp.wgred;
    if (!tail_combine) {
        TRY_HIP(launch_wgrad(wp, s), "conv weight gradient");
        return BNR_OK;
    }
    int64_t S = 1;
    TRY_HIP(launch_wgrad(wp, s, &S), "conv weight gradient");
    if (S > 1) {
        TRY_HIP(launch_bwd_tail(cp.wg, S, (int64_t)d->k * d->k * d->c_in * d->c_out, dw, cp.part, R, d->c_in, m,
                                dbeta, dgamma, split, s),
                "weight-gradient sum + backward sums combine");
    } else {
        TRY_HIP(launch_stats_finalize(cp.part, R, d->c_in, m, FIN_BWD, 0.f, nullptr, nullptr, nullptr, dbeta, dgamma,
                                      cp.red, s, split),
                "backward sums combine");
    }
    return BNR_OK;
}

// byte ranges a gradient source reads
static bool grad_src_overlaps(const bnr_conv_desc *d, const bnr_grad_src *g, Range r)
{
    const int es = esize(d->dtype);
    const int64_t m = pixels(d);
    if (g->kind == BNR_GRAD_DENSE || g->kind == BNR_GRAD_SPLIT)
        if (overlap(r, view_range(g->g, m, d->c_out, g->g_ldc, es))) return true;
    if (g->kind == BNR_GRAD_AVGPOOL2 && overlap(r, view_range(g->g, m / 4, d->c_out, g->g_ldc, es))) return true;
    if (g->kind == BNR_GRAD_BN && overlap(r, view_range(g->dy, m, d->c_out, d->c_out, es))) return true;
    if ((g->kind == BNR_GRAD_BN || g->kind == BNR_GRAD_SPLIT) && overlap(r, view_range(g->x, m, d->c_out, g->x_ldc, es)))
        return true;
    return false;
}

static bnr_status bwd_fused(const bnr_conv_desc *d, const void *x, const bnr_bn *x_bn, const void *w,
                            const bnr_grad_src *g, float *dw, float *dgamma, float *dbeta, void *dy, void *dx,
                            int32_t dx_ldc, int32_t dx_accumulate, void *ws, size_t ws_bytes, void *stream, int parts,
                            const void *z = nullptr, int32_t z_ldc = 0)
{
    TRY(check_desc(d));
    TRY(check_ptr(x, "x"));
    TRY(check_ptr(w, "w"));
    TRY(validate_grad_src(d, g));
    if (parts & BWD_WEIGHTS) TRY(check_fptr(dw, "dw"));
    if (x_bn) {
        TRY(check_bn(x_bn, "x_bn", true, false));
        TRY(check_fptr(dgamma, "dgamma"));
        TRY(check_fptr(dbeta, "dbeta"));
        TRY(check_ptr(dy, "dy"));
    } else if (!dx) {
        return fail(BNR_ERR_NULL, "dx is required when x_bn is NULL");
    }
    if (dx) {
        TRY(check_ptr(dx, "dx"));
        TRY(check_channels(d->c_in, dx_ldc, d->dtype, "dx"));
    }
    const ConvWs cw = conv_ws(d);
    TRY(check_ws(ws, ws_bytes, cw.total));
    const int es = esize(d->dtype);
    const int64_t m = pixels(d);
    const Range rx = view_range(x, m, d->c_in, d->in_ldc, es);
    // the data gradient's workgroups read every view of g_src while others
    // already write dy / dx, and the weight gradient reads them again: an
    // output overlapping any of them is an inter-workgroup race
    if (x_bn) {
        const Range rdy = view_range(dy, m, d->c_in, d->c_in, es);
        if (overlap(rdy, rx)) return fail(BNR_ERR_ALIAS, "dy overlaps x");
        if (grad_src_overlaps(d, g, rdy)) return fail(BNR_ERR_ALIAS, "dy overlaps a view g_src reads");
        if (dx && overlap(view_range(dx, m, d->c_in, dx_ldc, es), rx)) return fail(BNR_ERR_ALIAS, "dx overlaps x");
        if (dx && overlap(view_range(dx, m, d->c_in, dx_ldc, es), rdy)) return fail(BNR_ERR_ALIAS, "dx overlaps dy");
    }
    if (dx) {
        const Range rdx = view_range(dx, m, d->c_in, dx_ldc, es);
        if (grad_src_overlaps(d, g, rdx)) return fail(BNR_ERR_ALIAS, "dx overlaps a view g_src reads");
        if (!x_bn && overlap(rdx, rx)) return fail(BNR_ERR_ALIAS, "dx overlaps x");
    }
    if (z) {
        if (!x_bn) return fail(BNR_ERR_NULL, "z needs x_bn");
        TRY(check_ptr(z, "z"));
        TRY(check_channels(d->c_in, z_ldc, d->dtype, "z"));
        const Range rz = view_range(z, m, d->c_in, z_ldc, es);
        if (overlap(rz, view_range(dy, m, d->c_in, d->c_in, es)) ||
            (dx && overlap(rz, view_range(dx, m, d->c_in, dx_ldc, es))))
            return fail(BNR_ERR_ALIAS, "z overlaps dy or dx");
    }

    hipStream_t s = (hipStream_t)stream;
    if (x_bn) TRY(bwd_steps(d, x, x_bn, w, g, dw, dgamma, dbeta, dy, d->c_in, 0, 0, nullptr, ws, s, parts, z, z_ldc));
    else TRY(bwd_steps(d, x, nullptr, w, g, dw, nullptr, nullptr, dx, dx_ldc, 0, dx_accumulate, nullptr, ws, s, parts));
    // 4. optional standalone BN input gradient
    if ((parts & BWD_DATA) && x_bn && dx) {
        const Centred cx = centred(x_bn, dt_of(d->dtype));
        TRY_HIP(launch_elementwise(dt_of(d->dtype), EW_DX, m, d->c_in, dy, d->c_in, x, d->in_ldc, x_bn->gamma, nullptr,
                                   cx.mean, x_bn->rstd, dgamma, dbeta, dx, dx_ldc, dx_accumulate ? 1 : 0, s, cx.ctr),
                "BN input gradient");
    }
    return ok();
}

bnr_status bnr_bwd_fused(const bnr_conv_desc *d, const void *x, const bnr_bn *x_bn, const void *w,
                         const bnr_grad_src *g, float *dw, float *dgamma, float *dbeta, void *dy, void *dx,
                         int32_t dx_ldc, int32_t dx_accumulate, void *ws, size_t ws_bytes, void *stream)
{
    return bwd_fused(d, x, x_bn, w, g, dw, dgamma, dbeta, dy, dx, dx_ldc, dx_accumulate, ws, ws_bytes, stream,
                     BWD_DATA | BWD_WEIGHTS);
}

bnr_status bnr_bwd_fused_o2(const bnr_conv_desc *d, const void *x, const bnr_bn *x_bn, const void *z, int32_t z_ldc,
                            const void *w, const bnr_grad_src *g, float *dw, float *dgamma, float *dbeta, void *dy,
                            void *dx, int32_t dx_ldc, int32_t dx_accumulate, void *ws, size_t ws_bytes, void *stream)
{
    if (!x_bn) return fail(BNR_ERR_NULL, "x_bn is NULL");
    if (!z) return fail(BNR_ERR_NULL, "z is NULL");
    return bwd_fused(d, x, x_bn, w, g, dw, dgamma, dbeta, dy, dx, dx_ldc, dx_accumulate, ws, ws_bytes, stream,
                     BWD_DATA | BWD_WEIGHTS, z, z_ldc);
}

bnr_status bnr_bwd_data(const bnr_conv_desc *d, const void *x, const bnr_bn *x_bn, const void *w,
                        const bnr_grad_src *g, float *dgamma, float *dbeta, void *dy, void *dx, int32_t dx_ldc,
                        int32_t dx_accumulate, void *ws, size_t ws_bytes, void *stream)
{
    return bwd_fused(d, x, x_bn, w, g, nullptr, dgamma, dbeta, dy, dx, dx_ldc, dx_accumulate, ws, ws_bytes, stream,
                     BWD_DATA);
}

static bnr_status bwd_split(const bnr_conv_desc *d, const void *x, const bnr_bn *x_bn, const void *w,
                            const bnr_grad_src *g, float *dw, float *dgamma, float *dbeta, void *gsum,
                            int32_t gsum_ldc, int32_t accumulate, float *alpha, float *betap, void *ws,
                            size_t ws_bytes, void *stream, int parts)
{
    TRY(check_desc(d));
    TRY(check_ptr(x, "x"));
    TRY(check_ptr(w, "w"));
    TRY(validate_grad_src(d, g));
    if (parts & BWD_WEIGHTS) TRY(check_fptr(dw, "dw"));
    TRY(check_bn(x_bn, "x_bn", true, false));
    TRY(check_fptr(dgamma, "dgamma"));
    TRY(check_fptr(dbeta, "dbeta"));
    TRY(check_fptr(alpha, "alpha"));
    TRY(check_fptr(betap, "betap"));
    TRY(check_ptr(gsum, "gsum"));
    TRY(check_channels(d->c_in, gsum_ldc, d->dtype, "gsum"));
    const ConvWs cw = conv_ws(d);
    TRY(check_ws(ws, ws_bytes, cw.total));
    const int es = esize(d->dtype);
    const int64_t m = pixels(d);
    const Range rs = view_range(gsum, m, d->c_in, gsum_ldc, es);
    if (overlap(rs, view_range(x, m, d->c_in, d->in_ldc, es))) return fail(BNR_ERR_ALIAS, "gsum overlaps x");
    if (grad_src_overlaps(d, g, rs)) return fail(BNR_ERR_ALIAS, "gsum overlaps a view g_src reads");
    const SplitTerms st{x_bn->gamma, x_bn->rstd, alpha, betap, accumulate ? 1 : 0};
    TRY(bwd_steps(d, x, x_bn, w, g, dw, dgamma, dbeta, gsum, gsum_ldc, 1, accumulate ? 1 : 0, &st, ws,
                  (hipStream_t)stream, parts));
    return ok();
}

bnr_status bnr_bwd_fused_split(const bnr_conv_desc *d, const void *x, const bnr_bn *x_bn, const void *w,
                               const bnr_grad_src *g, float *dw, float *dgamma, float *dbeta, void *gsum,
                               int32_t gsum_ldc, int32_t accumulate, float *alpha, float *betap, void *ws,
                               size_t ws_bytes, void *stream)
{
    return bwd_split(d, x, x_bn, w, g, dw, dgamma, dbeta, gsum, gsum_ldc, accumulate, alpha, betap, ws, ws_bytes,
                     stream, BWD_DATA | BWD_WEIGHTS);
}

bnr_status bnr_bwd_data_split(const bnr_conv_desc *d, const void *x, const bnr_bn *x_bn, const void *w,
                              const bnr_grad_src *g, float *dgamma, float *dbeta, void *gsum, int32_t gsum_ldc,
                              int32_t accumulate, float *alpha, float *betap, void *ws, size_t ws_bytes,
                              void *stream)
{
    return bwd_split(d, x, x_bn, w, g, nullptr, dgamma, dbeta, gsum, gsum_ldc, accumulate, alpha, betap, ws,
                     ws_bytes, stream, BWD_DATA);
}

bnr_status bnr_bwd_weights(const bnr_conv_desc *d, const void *x, const bnr_bn *x_bn, const bnr_grad_src *g,
                           float *dw, void *ws, size_t ws_bytes, void *stream)
{
    TRY(check_desc(d));
    TRY(check_ptr(x, "x"));
    TRY(validate_grad_src(d, g));
    TRY(check_fptr(dw, "dw"));
    if (x_bn) TRY(check_bn(x_bn, "x_bn", true, false));
    const ConvWs cw = conv_ws(d);
    TRY(check_ws(ws, ws_bytes, cw.total));
    TRY(bwd_steps(d, x, x_bn, nullptr, g, dw, nullptr, nullptr, nullptr, 0, 0, 0, nullptr, ws, (hipStream_t)stream,
                  BWD_WEIGHTS));
    return ok();
}

bnr_status bnr_split_dx(int64_t m, int32_t c, bnr_dtype dtype, const void *gsum, int32_t gsum_ldc, const void *x,
                        int32_t x_ldc, const bnr_bn *bn, const float *alpha, const float *betap, void *dx,
                        int32_t dx_ldc, int32_t dx_accumulate, void *stream)
{
    TRY(check_dtype(dtype));
    if (m <= 0 || m > ((int64_t)1 << 31)) return fail(BNR_ERR_SHAPE, "m = %lld out of range", (long long)m);
    TRY(check_channels(c, gsum_ldc, dtype, "gsum"));
    TRY(check_channels(c, x_ldc, dtype, "x"));
    TRY(check_channels(c, dx_ldc, dtype, "dx"));
    TRY(check_ptr(gsum, "gsum"));
    TRY(check_ptr(x, "x"));
    TRY(check_ptr(dx, "dx"));
    TRY(check_bn(bn, "bn", false, false));
    TRY(check_fptr(alpha, "alpha"));
    TRY(check_fptr(betap, "betap"));
    const int es = esize(dtype);
    const Range rdx = view_range(dx, m, c, dx_ldc, es);
    if (overlap(rdx, view_range(x, m, c, x_ldc, es))) return fail(BNR_ERR_ALIAS, "dx overlaps x");
    if (overlap(rdx, view_range(gsum, m, c, gsum_ldc, es)) && !(gsum == dx && dx_ldc == gsum_ldc && !dx_accumulate))
        return fail(BNR_ERR_ALIAS, "dx overlaps gsum");
    const Centred cx = centred(bn, dt_of(dtype));
    TRY_HIP(launch_elementwise(dt_of(dtype), EW_SPLITDX, m, c, gsum, gsum_ldc, x, x_ldc, nullptr, nullptr, cx.mean,
                               bn->rstd, betap, alpha, dx, dx_ldc, dx_accumulate ? 1 : 0, (hipStream_t)stream, cx.ctr),
            "summed BN input gradient");
    return ok();
}

bnr_status bnr_bn_dx(int64_t m, int32_t c, bnr_dtype dtype, const void *dy, const void *x, int32_t x_ldc,
                     const bnr_bn *bn, const float *dgamma, const float *dbeta, void *dx, int32_t dx_ldc,
                     int32_t dx_accumulate, void *stream)
{
    TRY(check_dtype(dtype));
    if (m <= 0 || m > ((int64_t)1 << 31)) return fail(BNR_ERR_SHAPE, "m = %lld out of range", (long long)m);
    TRY(check_channels(c, c, dtype, "dy"));
    TRY(check_channels(c, x_ldc, dtype, "x"));
    TRY(check_channels(c, dx_ldc, dtype, "dx"));
    TRY(check_ptr(dy, "dy"));
    TRY(check_ptr(x, "x"));
    TRY(check_ptr(dx, "dx"));
    TRY(check_bn(bn, "bn", true, false));
    TRY(check_fptr(dgamma, "dgamma"));
    TRY(check_fptr(dbeta, "dbeta"));
    const int es = esize(dtype);
    const Range rdx = view_range(dx, m, c, dx_ldc, es);
    if (overlap(rdx, view_range(x, m, c, x_ldc, es))) return fail(BNR_ERR_ALIAS, "dx overlaps x");
    const Range rdy = view_range(dy, m, c, c, es);
    if (overlap(rdx, rdy) && !(dy == dx && dx_ldc == c && !dx_accumulate))
        return fail(BNR_ERR_ALIAS, "dx overlaps dy");
    const Centred cx = centred(bn, dt_of(dtype));
    TRY_HIP(launch_elementwise(dt_of(dtype), EW_DX, m, c, dy, c, x, x_ldc, bn->gamma, nullptr, cx.mean, bn->rstd,
                               dgamma, dbeta, dx, dx_ldc, dx_accumulate ? 1 : 0, (hipStream_t)stream, cx.ctr),
            "BN input gradient");
    return ok();
}

bnr_status bnr_reference_path(bnr_ref_mode mode, int32_t backward, const bnr_conv_desc *d, const bnr_ref_args *a,
                              void *ws, size_t ws_bytes, void *stream)
{
    TRY(check_desc(d));
    if (mode != BNR_MODE_BASELINE && mode != BNR_MODE_RCF && mode != BNR_MODE_RCF_MVF)
        return fail(BNR_ERR_UNSUPPORTED, "unknown reference mode %d", (int)mode);
    if (!a) return fail(BNR_ERR_NULL, "args is NULL");
    const bool base = mode == BNR_MODE_BASELINE;
    TRY(check_ptr(a->x, "x"));
    TRY(check_ptr(a->w, "w"));
    TRY(check_ptr(a->y, "y"));
    if (base) TRY(check_ptr(a->z, "z"));
    TRY(check_bn(a->bn, "bn", true, !backward));
    const ConvWs cw = conv_ws(d);
    TRY(check_ws(ws, ws_bytes, cw.total));
    const int64_t m = pixels(d);
    const int es = esize(d->dtype);
    const int dt = dt_of(d->dtype);
    hipStream_t s = (hipStream_t)stream;
    const ConvPtrs cp = conv_ptrs(ws, cw);
    void *wpack = cp.pack;
    float *part = cp.part;
    void *red = cp.red;
    const bnr_bn *bn = a->bn;

    if (!backward) {
        TRY(check_ptr(a->out, "out"));
        if (overlap(view_range(a->out, m, d->c_out, d->out_ldc, es), view_range(a->x, m, d->c_in, d->in_ldc, es)))
            return fail(BNR_ERR_ALIAS, "out overlaps x");
        const int64_t R = stats_row_blocks(m, d->c_in, dt);
        if (mode == BNR_MODE_RCF_MVF) {
            TRY_HIP(launch_stats_partial(dt, a->x, d->in_ldc, m, d->c_in, ST_SUMSQ, bn->shift, nullptr, nullptr, 0,
                                         part, R, s), "stats sweep");
            const SplitTerms ft = fwd_terms(bn, true);
            TRY_HIP(launch_stats_finalize(part, R, d->c_in, m, FIN_MVF, bn->eps, bn->mean, bn->var, bn->rstd,
                                          nullptr, nullptr, red, s, &ft), "stats combine");
        } else {
            // mean sweep, then variance sweep (two-pass, as the unfused BN layer)
            TRY_HIP(launch_stats_partial(dt, a->x, d->in_ldc, m, d->c_in, ST_SUM, nullptr, nullptr, nullptr, 0, part,
                                         R, s), "mean sweep");
            const SplitTerms mt = mean_terms(bn);
            TRY_HIP(launch_stats_finalize(part, R, d->c_in, m, FIN_MEAN, bn->eps, bn->mean, nullptr, nullptr, nullptr,
                                          nullptr, red, s, &mt), "mean combine");
            TRY_HIP(launch_stats_partial(dt, a->x, d->in_ldc, m, d->c_in, ST_SQDEV, bn->mean, nullptr, nullptr, 0,
                                         part, R, s), "variance sweep");
            const SplitTerms ft = fwd_terms(bn, false);
            TRY_HIP(launch_stats_finalize(part, R, d->c_in, m, FIN_VAR, bn->eps, bn->mean, bn->var, bn->rstd, nullptr,
                                          nullptr, red, s, &ft), "variance combine");
        }
        const Centred cx = centred(bn, dt);
        TRY_HIP(launch_elementwise(dt, EW_APPLY, m, d->c_in, a->x, d->in_ldc, nullptr, 0, bn->gamma, bn->beta,
                                   cx.mean, bn->rstd, nullptr, nullptr, a->y, d->c_in, 0, s, cx.ctr), "normalise");
        if (base)
            TRY_HIP(launch_elementwise(dt, EW_RELU, m, d->c_in, a->y, d->c_in, nullptr, 0, nullptr, nullptr, nullptr,
                                       nullptr, nullptr, nullptr, a->z, d->c_in, 0, s), "relu");
        RowsParams rp;
        fill_rows(rp, d, d->c_in, d->c_out);
        rp.pro = base ? PRO_NONE : PRO_RELU;
        rp.a = base ? a->z : a->y; rp.a_ldc = d->c_in;
        rp.epi = EPI_STORE; rp.y = a->out; rp.y_ldc = d->out_ldc;
        int64_t Rf = 0;
        TRY(launch_conv_any(rp, d, a->w, 0, wpack, &Rf, s));
        return ok();
    }

    TRY(check_ptr(a->g, "g"));
    TRY(check_channels(d->c_out, a->g_ldc, d->dtype, "g"));
    if (base) TRY(check_ptr(a->dz, "dz"));
    TRY(check_ptr(a->dy, "dy"));
    TRY(check_fptr(a->dw, "dw"));
    TRY(check_fptr(a->dgamma, "dgamma"));
    TRY(check_fptr(a->dbeta, "dbeta"));
    TRY(check_ptr(a->dx, "dx"));
    TRY(check_channels(d->c_in, a->dx_ldc, d->dtype, "dx"));
    if (overlap(view_range(a->dx, m, d->c_in, a->dx_ldc, es), view_range(a->x, m, d->c_in, d->in_ldc, es)))
        return fail(BNR_ERR_ALIAS, "dx overlaps x");
    // data gradient (BASELINE: materialise dz; RCF: ReLU mask in the epilogue)
    RowsParams rp;
    fill_rows(rp, d, d->c_out, d->c_in);
    rp.pro = PRO_NONE; rp.a = a->g; rp.a_ldc = a->g_ldc;
    if (base) {
        rp.epi = EPI_STORE; rp.y = a->dz; rp.y_ldc = d->c_in;
    } else {
        rp.epi = EPI_RELUMASK; rp.y = a->dy; rp.y_ldc = d->c_in; rp.ex = a->y; rp.ex_ldc = d->c_in;
    }
    int64_t Rd = 0;
    TRY(launch_conv_any(rp, d, a->w, 1, wpack, &Rd, s));
    // weight gradient (BASELINE reads the stored z; RCF recomputes relu(y))
    WgradParams wp;
    memset(&wp, 0, sizeof wp);
    wp.dtype = dt; wp.k = d->k; wp.n = d->n; wp.h = d->h; wp.w = d->w; wp.m = m;
    wp.c_in = d->c_in; wp.c_out = d->c_out;
    wp.x = base ? a->z : a->y; wp.x_ldc = d->c_in; wp.a_mode = base ? 0 : 2;
    wp.gsrc = GB_DENSE; wp.g = a->g; wp.g_ldc = a->g_ldc;
    wp.dw = a->dw; wp.part = cp.wg; wp.red = cp.wgred;
    TRY_HIP(launch_wgrad(wp, s), "conv weight gradient");
    if (base)
        TRY_HIP(launch_elementwise(dt, EW_RELUBWD, m, d->c_in, a->dz, d->c_in, a->y, d->c_in, nullptr, nullptr, nullptr,
                                   nullptr, nullptr, nullptr, a->dy, d->c_in, 0, s), "relu backward");
    const int64_t R = stats_row_blocks(m, d->c_in, dt);
    const Centred cx = centred(bn, dt);
    TRY_HIP(launch_stats_partial(dt, a->x, d->in_ldc, m, d->c_in, ST_DYX, cx.mean, bn->rstd, a->dy, d->c_in, part, R,
                                 s, cx.ctr), "BN backward sums sweep");
    TRY_HIP(launch_stats_finalize(part, R, d->c_in, m, FIN_BWD, 0.f, nullptr, nullptr, nullptr, a->dbeta, a->dgamma,
                                  red, s),
            "BN backward sums combine");
    TRY_HIP(launch_elementwise(dt, EW_DX, m, d->c_in, a->dy, d->c_in, a->x, d->in_ldc, bn->gamma, nullptr, cx.mean,
                               bn->rstd, a->dgamma, a->dbeta, a->dx, a->dx_ldc, a->dx_accumulate ? 1 : 0, s, cx.ctr),
            "BN input gradient");
    return ok();
}

bnr_status bnr_conv_fwd(const bnr_conv_desc *d, const void *x, const void *w, void *y, void *ws, size_t ws_bytes,
                        void *stream)
{
    return conv_fwd(d, x, nullptr, w, y, nullptr, ws, ws_bytes, stream);
}

// shared argument checks of the residual BN-add-ReLU calls
static bnr_status check_rows(int64_t m, int32_t c, bnr_dtype dtype)
{
    TRY(check_dtype(dtype));
    if (m <= 0 || m > ((int64_t)1 << 31)) return fail(BNR_ERR_SHAPE, "m = %lld out of range", (long long)m);
    return check_channels(c, c, dtype, "c");
}

bnr_status bnr_bn_add_relu_fwd(int64_t m, int32_t c, bnr_dtype dtype, const void *y, int32_t y_ldc, const bnr_bn *bn,
                               const void *id, int32_t id_ldc, void *out, int32_t out_ldc, void *stream)
{
    TRY(check_rows(m, c, dtype));
    TRY(check_channels(c, y_ldc, dtype, "y"));
    TRY(check_channels(c, id_ldc, dtype, "id"));
    TRY(check_channels(c, out_ldc, dtype, "out"));
    TRY(check_ptr(y, "y"));
    TRY(check_ptr(id, "id"));
    TRY(check_ptr(out, "out"));
    TRY(check_bn(bn, "bn", true, false));
    const int es = esize(dtype);
    const Range ro = view_range(out, m, c, out_ldc, es);
    if (overlap(ro, view_range(y, m, c, y_ldc, es))) return fail(BNR_ERR_ALIAS, "out overlaps y");
    if (overlap(ro, view_range(id, m, c, id_ldc, es)) && !(out == id && out_ldc == id_ldc))
        return fail(BNR_ERR_ALIAS, "out overlaps id");
    const Centred cy = centred(bn, dt_of(dtype));
    TRY_HIP(launch_elementwise(dt_of(dtype), EW_BNADDRELU, m, c, y, y_ldc, id, id_ldc, bn->gamma, bn->beta, cy.mean,
                               bn->rstd, nullptr, nullptr, out, out_ldc, 0, (hipStream_t)stream, cy.ctr),
            "BN + add + ReLU");
    return ok();
}

bnr_status bnr_bn_add_relu_bwd(int64_t m, int32_t c, bnr_dtype dtype, const void *g, int32_t g_ldc, const void *out,
                               int32_t out_ldc, const void *y, int32_t y_ldc, const bnr_bn *bn, void *gm,
                               int32_t gm_ldc, float *dgamma, float *dbeta, void *ws, size_t ws_bytes, void *stream)
{
    TRY(check_rows(m, c, dtype));
    TRY(check_channels(c, g_ldc, dtype, "g"));
    TRY(check_channels(c, out_ldc, dtype, "out"));
    TRY(check_channels(c, y_ldc, dtype, "y"));
    TRY(check_channels(c, gm_ldc, dtype, "gm"));
    TRY(check_ptr(g, "g"));
    TRY(check_ptr(out, "out"));
    TRY(check_ptr(y, "y"));
    TRY(check_ptr(gm, "gm"));
    TRY(check_bn(bn, "bn", false, false));
    TRY(check_fptr(dgamma, "dgamma"));
    TRY(check_fptr(dbeta, "dbeta"));
    TRY(check_ws(ws, ws_bytes, stats_ws(m, c)));
    const int es = esize(dtype);
    const Range rg = view_range(gm, m, c, gm_ldc, es);
    if (overlap(rg, view_range(out, m, c, out_ldc, es))) return fail(BNR_ERR_ALIAS, "gm overlaps out");
    if (overlap(rg, view_range(y, m, c, y_ldc, es))) return fail(BNR_ERR_ALIAS, "gm overlaps y");
    if (overlap(rg, view_range(g, m, c, g_ldc, es)) && !(gm == g && gm_ldc == g_ldc))
        return fail(BNR_ERR_ALIAS, "gm overlaps g");
    hipStream_t s = (hipStream_t)stream;
    const int dt = dt_of(dtype);
    const int64_t R = stats_row_blocks(m, c, dt);
    float *part = (float *)ws;
    void *red = (char *)ws + stats_part_bytes(m, c);
    const Centred cy = centred(bn, dt);
    TRY_HIP(launch_addrelu_bwd(dt, m, c, g, g_ldc, out, out_ldc, y, y_ldc, cy.mean, bn->rstd, gm, gm_ldc, part, R, s,
                               cy.ctr),
            "ReLU mask + BN backward sums");
    TRY_HIP(launch_stats_finalize(part, R, c, m, FIN_BWD, 0.f, nullptr, nullptr, nullptr, dbeta, dgamma, red, s),
            "backward sums combine");
    return ok();
}

bnr_status bnr_reference_bn_add_relu(int32_t backward, int64_t m, int32_t c, bnr_dtype dtype,
                                     const bnr_addrelu_ref_args *a, void *ws, size_t ws_bytes, void *stream)
{
    TRY(check_rows(m, c, dtype));
    if (!a) return fail(BNR_ERR_NULL, "args is NULL");
    TRY(check_channels(c, a->y_ldc, dtype, "y"));
    TRY(check_ptr(a->y, "y"));
    TRY(check_ptr(a->out, "out"));
    TRY(check_channels(c, a->out_ldc, dtype, "out"));
    TRY(check_ws(ws, ws_bytes, stats_ws(m, c)));
    hipStream_t s = (hipStream_t)stream;
    const int dt = dt_of(dtype);
    const bnr_bn *bn = a->bn;
    const int64_t R = stats_row_blocks(m, c, dt);
    float *part = (float *)ws;
    void *red = (char *)ws + stats_part_bytes(m, c);
    if (!backward) {
        TRY(check_bn(bn, "bn", true, true));
        TRY(check_ptr(a->id, "id"));
        TRY(check_channels(c, a->id_ldc, dtype, "id"));
        TRY(check_ptr(a->tmp, "tmp"));
        // two-pass statistics, normalise (write tmp), add + ReLU (write out)
        TRY_HIP(launch_stats_partial(dt, a->y, a->y_ldc, m, c, ST_SUM, nullptr, nullptr, nullptr, 0, part, R, s),
                "mean sweep");
        const SplitTerms mt = mean_terms(bn);
        TRY_HIP(launch_stats_finalize(part, R, c, m, FIN_MEAN, bn->eps, bn->mean, nullptr, nullptr, nullptr, nullptr,
                                      red, s, &mt), "mean combine");
        TRY_HIP(launch_stats_partial(dt, a->y, a->y_ldc, m, c, ST_SQDEV, bn->mean, nullptr, nullptr, 0, part, R, s),
                "variance sweep");
        const SplitTerms ft = fwd_terms(bn, false);
        TRY_HIP(launch_stats_finalize(part, R, c, m, FIN_VAR, bn->eps, bn->mean, bn->var, bn->rstd, nullptr, nullptr,
                                      red, s, &ft), "variance combine");
        const Centred cy = centred(bn, dt);
        TRY_HIP(launch_elementwise(dt, EW_APPLY, m, c, a->y, a->y_ldc, nullptr, 0, bn->gamma, bn->beta, cy.mean,
                                   bn->rstd, nullptr, nullptr, a->tmp, c, 0, s, cy.ctr), "normalise");
        TRY_HIP(launch_elementwise(dt, EW_ADDRELU, m, c, a->tmp, c, a->id, a->id_ldc, nullptr, nullptr, nullptr,
                                   nullptr, nullptr, nullptr, a->out, a->out_ldc, 0, s), "add + ReLU");
        return ok();
    }
    TRY(check_bn(bn, "bn", true, false));
    TRY(check_ptr(a->g, "g"));
    TRY(check_channels(c, a->g_ldc, dtype, "g"));
    TRY(check_ptr(a->gm, "gm"));
    TRY(check_ptr(a->dx, "dx"));
    TRY(check_channels(c, a->dx_ldc, dtype, "dx"));
    TRY(check_fptr(a->dgamma, "dgamma"));
    TRY(check_fptr(a->dbeta, "dbeta"));
    // ReLU backward (write gm), BN reductions sweep, BN input-gradient sweep (write dx)
    TRY_HIP(launch_elementwise(dt, EW_RELUBWD, m, c, a->g, a->g_ldc, a->out, a->out_ldc, nullptr, nullptr, nullptr,
                               nullptr, nullptr, nullptr, a->gm, c, 0, s), "ReLU backward");
    const Centred cy = centred(bn, dt);
    TRY_HIP(launch_stats_partial(dt, a->y, a->y_ldc, m, c, ST_DYX, cy.mean, bn->rstd, a->gm, c, part, R, s, cy.ctr),
            "BN backward sums");
    TRY_HIP(launch_stats_finalize(part, R, c, m, FIN_BWD, 0.f, nullptr, nullptr, nullptr, a->dbeta, a->dgamma, red, s),
            "backward sums combine");
    TRY_HIP(launch_elementwise(dt, EW_DX, m, c, a->gm, c, a->y, a->y_ldc, bn->gamma, nullptr, cy.mean, bn->rstd,
                               a->dgamma, a->dbeta, a->dx, a->dx_ldc, 0, s, cy.ctr), "BN input gradient");
    return ok();
}

bnr_status bnr_reference_bn_relu(int32_t backward, int64_t m, int32_t c, bnr_dtype dtype, const bnr_bnrelu_ref_args *a,
                                 void *ws, size_t ws_bytes, void *stream)
{
    TRY(check_rows(m, c, dtype));
    if (!a) return fail(BNR_ERR_NULL, "args is NULL");
    TRY(check_channels(c, a->x_ldc, dtype, "x"));
    TRY(check_ptr(a->x, "x"));
    TRY(check_ptr(a->y, "y"));
    TRY(check_ws(ws, ws_bytes, stats_ws(m, c)));
    const int es = esize(dtype);
    hipStream_t s = (hipStream_t)stream;
    const int dt = dt_of(dtype);
    const bnr_bn *bn = a->bn;
    const int64_t R = stats_row_blocks(m, c, dt);
    float *part = (float *)ws;
    void *red = (char *)ws + stats_part_bytes(m, c);
    const Range rx = view_range(a->x, m, c, a->x_ldc, es), ry = view_range(a->y, m, c, c, es);
    if (overlap(rx, ry)) return fail(BNR_ERR_ALIAS, "y overlaps x");
    if (!backward) {
        TRY(check_bn(bn, "bn", true, true));
        TRY(check_ptr(a->z, "z"));
        const Range rz = view_range(a->z, m, c, c, es);
        if (overlap(rz, rx) || overlap(rz, ry)) return fail(BNR_ERR_ALIAS, "z overlaps x or y");
        // two-pass statistics, normalise (write y), ReLU (write z)
        TRY_HIP(launch_stats_partial(dt, a->x, a->x_ldc, m, c, ST_SUM, nullptr, nullptr, nullptr, 0, part, R, s),
                "mean sweep");
        const SplitTerms mt = mean_terms(bn);
        TRY_HIP(launch_stats_finalize(part, R, c, m, FIN_MEAN, bn->eps, bn->mean, nullptr, nullptr, nullptr, nullptr,
                                      red, s, &mt), "mean combine");
        TRY_HIP(launch_stats_partial(dt, a->x, a->x_ldc, m, c, ST_SQDEV, bn->mean, nullptr, nullptr, 0, part, R, s),
                "variance sweep");
        const SplitTerms ft = fwd_terms(bn, false);
        TRY_HIP(launch_stats_finalize(part, R, c, m, FIN_VAR, bn->eps, bn->mean, bn->var, bn->rstd, nullptr, nullptr,
                                      red, s, &ft), "variance combine");
        const Centred cx = centred(bn, dt);
        TRY_HIP(launch_elementwise(dt, EW_APPLY, m, c, a->x, a->x_ldc, nullptr, 0, bn->gamma, bn->beta, cx.mean,
                                   bn->rstd, nullptr, nullptr, a->y, c, 0, s, cx.ctr), "normalise");
        TRY_HIP(launch_elementwise(dt, EW_RELU, m, c, a->y, c, nullptr, 0, nullptr, nullptr, nullptr, nullptr, nullptr,
                                   nullptr, a->z, c, 0, s), "ReLU");
        return ok();
    }
    TRY(check_bn(bn, "bn", true, false));
    TRY(check_ptr(a->gz, "gz"));
    TRY(check_channels(c, a->gz_ldc, dtype, "gz"));
    TRY(check_ptr(a->dy, "dy"));
    TRY(check_ptr(a->dx, "dx"));
    TRY(check_channels(c, a->dx_ldc, dtype, "dx"));
    TRY(check_fptr(a->dgamma, "dgamma"));
    TRY(check_fptr(a->dbeta, "dbeta"));
    const Range rd = view_range(a->dy, m, c, c, es), rdx = view_range(a->dx, m, c, a->dx_ldc, es);
    if (overlap(rd, rx) || overlap(rd, ry) || overlap(rdx, rx) || overlap(rdx, ry) || overlap(rdx, rd))
        return fail(BNR_ERR_ALIAS, "dy / dx overlap an input");
    // ReLU backward (write dy), BN reductions sweep, BN input-gradient sweep (write dx)
    TRY_HIP(launch_elementwise(dt, EW_RELUBWD, m, c, a->gz, a->gz_ldc, a->y, c, nullptr, nullptr, nullptr, nullptr,
                               nullptr, nullptr, a->dy, c, 0, s), "ReLU backward");
    const Centred cx = centred(bn, dt);
    TRY_HIP(launch_stats_partial(dt, a->x, a->x_ldc, m, c, ST_DYX, cx.mean, bn->rstd, a->dy, c, part, R, s, cx.ctr),
            "BN backward sums");
    TRY_HIP(launch_stats_finalize(part, R, c, m, FIN_BWD, 0.f, nullptr, nullptr, nullptr, a->dbeta, a->dgamma, red, s),
            "backward sums combine");
    TRY_HIP(launch_elementwise(dt, EW_DX, m, c, a->dy, c, a->x, a->x_ldc, bn->gamma, nullptr, cx.mean, bn->rstd,
                               a->dgamma, a->dbeta, a->dx, a->dx_ldc, 0, s, cx.ctr), "BN input gradient");
    return ok();
}

bnr_status bnr_hbm_copy(const void *src, void *dst, size_t bytes, void *stream)
{
    TRY(check_ptr(src, "src"));
    TRY(check_ptr(dst, "dst"));
    if (bytes == 0 || bytes % 16) return fail(BNR_ERR_SHAPE, "bytes must be a positive multiple of 16");
    Range a{(uintptr_t)src, (uintptr_t)src + bytes}, b{(uintptr_t)dst, (uintptr_t)dst + bytes};
    if (overlap(a, b)) return fail(BNR_ERR_ALIAS, "dst overlaps src");
    TRY_HIP(launch_copy16(src, dst, (int64_t)(bytes / 16), (hipStream_t)stream), "copy");
    return ok();
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Network ends: first CONV, BN-ReLU-max pooling, classifier head.
namespace {

bnr_status check_stem(const bnr_stem_desc *d)
{
    if (!d) return fail(BNR_ERR_NULL, "desc is NULL");
    TRY(check_dtype(d->dtype));
    if (d->n <= 0 || d->h <= 0 || d->w <= 0) return fail(BNR_ERR_SHAPE, "n, h, w must be positive");
    if (d->c_in < 1 || d->c_in > kStemPix) return fail(BNR_ERR_UNSUPPORTED, "c_in %d (1..%d)", d->c_in, kStemPix);
    if (d->w > kStemMaxW) return fail(BNR_ERR_UNSUPPORTED, "image width %d > %d", d->w, kStemMaxW);
    if ((int64_t)d->n * d->h * d->w * kStemPix >= ((int64_t)1 << 31)) return fail(BNR_ERR_SHAPE, "image too large");
    if ((int64_t)d->n * stem_out(d->h) * stem_out(d->w) * kStemCout >= ((int64_t)1 << 31))
        return fail(BNR_ERR_SHAPE, "output too large");
    return BNR_OK;
}

struct StemWs { size_t part, red, wg, wgred, total; };
StemWs stem_ws(const bnr_stem_desc *d)
{
    const int ho = stem_out(d->h), wo = stem_out(d->w);
    const int64_t m = (int64_t)d->n * ho * wo;
    const int64_t items = (int64_t)d->n * ((ho + kStemRows - 1) / kStemRows);
    const int64_t nw = (int64_t)kStemK * kStemK * d->c_in * kStemCout;
    StemWs w;
    const size_t pg = (size_t)stem_groups(items) * 2 * kStemCout * 4, ps = stats_part_bytes(m, kStemCout);
    w.part = align_up(pg > ps ? pg : ps);
    w.red = align_up(stats_red_bytes(kStemCout));
    w.wg = align_up((size_t)stem_wgrad_splits(DT_BF16, items) * nw * 4);
    w.wgred = align_up(sum_partials_red_bytes(nw));
    w.total = w.part + w.red + w.wg + w.wgred;
    return w;
}

void stem_params(StemParams &p, const bnr_stem_desc *d)
{
    memset(&p, 0, sizeof p);
    p.n = d->n; p.h = d->h; p.w = d->w;
    p.ho = stem_out(d->h); p.wo = stem_out(d->w);
    p.c_in = d->c_in;
}

Range bytes_range(const void *p, int64_t bytes)
{
    const uintptr_t lo = reinterpret_cast<uintptr_t>(p);
    return Range{lo, lo + (uintptr_t)bytes};
}

size_t pool_ws(int n, int h, int w, int c)
{
    const int64_t m_out = (int64_t)n * ((h - 1) / 2 + 1) * ((w - 1) / 2 + 1);
    int64_t R = maxpool_fwd_rows(DT_BF16, m_out, c);
    if (maxpool_fwd_rows(DT_F32, m_out, c) > R) R = maxpool_fwd_rows(DT_F32, m_out, c);
    if (maxpool_bwd_groups(n, h) > R) R = maxpool_bwd_groups(n, h);
    return align_up((size_t)R * 2 * c * 4) + align_up(stats_red_bytes(c));
}

bnr_status check_pool_shape(int n, int h, int w, int c)
{
    if (n <= 0 || h <= 0 || w <= 0 || c <= 0) return fail(BNR_ERR_SHAPE, "n, h, w, c must be positive");
    if ((int64_t)n * h * w > ((int64_t)1 << 31)) return fail(BNR_ERR_SHAPE, "too many pixels");
    return BNR_OK;
}

size_t head_ws(int n, int h, int w, int c)
{
    const int64_t m = (int64_t)n * h * w;
    int64_t R = head_rows(DT_BF16, m, c);
    if (head_rows(DT_F32, m, c) > R) R = head_rows(DT_F32, m, c);
    return align_up((size_t)R * 2 * c * 4) + align_up(stats_red_bytes(c));
}

bnr_status check_head(int n, int h, int w, int c, int classes, bnr_dtype dtype, const void *x, int x_ldc,
                      const bnr_bn *x_bn, const void *wfc)
{
    TRY(check_dtype(dtype));
    if (n <= 0 || h <= 0 || w <= 0 || classes <= 0) return fail(BNR_ERR_SHAPE, "n, h, w, classes must be positive");
    if ((int64_t)n * h * w > ((int64_t)1 << 31) || (int64_t)c * classes > ((int64_t)1 << 31))
        return fail(BNR_ERR_SHAPE, "too large");
    TRY(check_channels(c, x_ldc, dtype, "x"));
    TRY(check_ptr(x, "x"));
    TRY(check_bn(x_bn, "x_bn", true, false));
    TRY(check_ptr(wfc, "wfc"));
    return BNR_OK;
}

void head_params(HeadParams &p, int dt, int n, int h, int w, int c, int classes, const void *x, int x_ldc,
                 const bnr_bn *bn, const void *wfc)
{
    memset(&p, 0, sizeof p);
    p.n = n; p.h = h; p.w = w; p.c = c; p.classes = classes;
    p.x = x; p.x_ldc = x_ldc;
    const Centred cx = centred(bn, dt);
    p.gamma = bn->gamma; p.beta = bn->beta; p.mean = cx.mean; p.rstd = bn->rstd; p.ctr = cx.ctr;
    p.wfc = wfc;
}

}  // namespace

extern "C" {

size_t bnr_stem_workspace_size(const bnr_stem_desc *d)
{
    if (check_stem(d) != BNR_OK) return 0;
    return stem_ws(d).total;
}

bnr_status bnr_stem_conv_fwd(const bnr_stem_desc *d, const void *img, const void *w, void *s, bnr_bn *s_bn, void *ws,
                             size_t ws_bytes, void *stream)
{
    TRY(check_stem(d));
    TRY(check_ptr(img, "img"));
    TRY(check_ptr(w, "w"));
    TRY(check_ptr(s, "s"));
    if (s_bn) TRY(check_bn(s_bn, "s_bn", false, true));
    const StemWs sw = stem_ws(d);
    TRY(check_ws(ws, ws_bytes, sw.total));
    const int es = esize(d->dtype);
    StemParams p;
    stem_params(p, d);
    const int64_t m = (int64_t)p.n * p.ho * p.wo;
    const Range rs = bytes_range(s, m * kStemCout * es);
    if (overlap(rs, bytes_range(img, (int64_t)d->n * d->h * d->w * kStemPix * es))) return fail(BNR_ERR_ALIAS, "s overlaps img");
    if (overlap(rs, bytes_range(w, (int64_t)kStemK * kStemK * d->c_in * kStemCout * es)))
        return fail(BNR_ERR_ALIAS, "s overlaps w");
    p.img = img; p.wt = w; p.s = s;
    p.part = (float *)ws;
    p.shift = s_bn ? s_bn->shift : nullptr;
    hipStream_t st = (hipStream_t)stream;
    const int dt = dt_of(d->dtype);
    TRY_HIP(launch_stem_conv(dt, p, s_bn && dt == DT_BF16, st), "first conv");
    if (s_bn) {
        if (dt == DT_BF16) {
            const int64_t R = stem_groups((int64_t)p.n * ((p.ho + kStemRows - 1) / kStemRows));
            const SplitTerms ft = fwd_terms(s_bn, true);
            TRY_HIP(launch_stats_finalize(p.part, R, kStemCout, m, FIN_MVF, s_bn->eps, s_bn->mean, s_bn->var,
                                          s_bn->rstd, nullptr, nullptr, (char *)ws + sw.part, st, &ft),
                    "stats combine");
        } else {
            TRY(run_stats(m, kStemCout, kStemCout, d->dtype, s, s_bn, ws, st));
        }
    }
    return ok();
}

bnr_status bnr_stem_wgrad(const bnr_stem_desc *d, const void *img, const bnr_grad_src *g, float *dw, void *ws,
                          size_t ws_bytes, void *stream)
{
    TRY(check_stem(d));
    TRY(check_ptr(img, "img"));
    TRY(check_ptr(dw, "dw"));
    if (!g) return fail(BNR_ERR_NULL, "g_src is NULL");
    StemParams p;
    stem_params(p, d);
    if (g->kind == BNR_GRAD_DENSE) {
        TRY(check_ptr(g->g, "g_src.g"));
        TRY(check_channels(kStemCout, g->g_ldc, d->dtype, "g_src.g"));
        p.g = g->g;
        p.g_ldc = g->g_ldc;
    } else if (g->kind == BNR_GRAD_BN) {
        TRY(check_ptr(g->dy, "g_src.dy"));
        TRY(check_ptr(g->x, "g_src.x"));
        TRY(check_channels(kStemCout, g->x_ldc, d->dtype, "g_src.x"));
        TRY(check_bn(g->bn, "g_src.bn", true, false));
        TRY(check_fptr(g->dgamma, "g_src.dgamma"));
        TRY(check_fptr(g->dbeta, "g_src.dbeta"));
        p.g = g->dy;
        p.g_ldc = kStemCout;
        p.gx = g->x;
        p.gx_ldc = g->x_ldc;
        const Centred cg = centred(g->bn, dt_of(d->dtype));
        p.g_gamma = g->bn->gamma; p.g_mean = cg.mean; p.g_rstd = g->bn->rstd; p.g_ctr = cg.ctr;
        p.g_dgamma = g->dgamma; p.g_dbeta = g->dbeta;
    } else {
        return fail(BNR_ERR_UNSUPPORTED, "gradient kind %d (first CONV: dense or BN)", (int)g->kind);
    }
    const StemWs sw = stem_ws(d);
    TRY(check_ws(ws, ws_bytes, sw.total));
    p.img = img;
    hipStream_t st = (hipStream_t)stream;
    const int dt = dt_of(d->dtype);
    const int gs = g->kind == BNR_GRAD_BN ? GB_BNGRAD : GB_DENSE;
    if (dt == DT_BF16) {
        const int64_t S = stem_wgrad_splits(dt, (int64_t)p.n * ((p.ho + kStemRows - 1) / kStemRows));
        const int64_t len = (int64_t)kStemK * kStemK * d->c_in * kStemCout;
        p.dwpart = (float *)((char *)ws + sw.part + sw.red);
        TRY_HIP(launch_stem_wgrad(dt, p, gs, st), "first conv weight gradient");
        TRY_HIP(launch_sum_partials(p.dwpart, S, len, dw, (char *)ws + sw.part + sw.red + sw.wg, st),
                "weight gradient split sum");
    } else {
        p.dwpart = dw;
        TRY_HIP(launch_stem_wgrad(dt, p, gs, st), "first conv weight gradient");
    }
    return ok();
}

size_t bnr_pool_workspace_size(int32_t n, int32_t h, int32_t w, int32_t c)
{
    if (check_pool_shape(n, h, w, c) != BNR_OK) return 0;
    return pool_ws(n, h, w, c);
}

bnr_status bnr_bn_relu_maxpool_fwd(int32_t n, int32_t h, int32_t w, int32_t c, bnr_dtype dtype, const void *x,
                                   int32_t x_ldc, const bnr_bn *x_bn, void *y, int32_t y_ldc, bnr_bn *y_bn, void *ws,
                                   size_t ws_bytes, void *stream)
{
    TRY(check_dtype(dtype));
    TRY(check_pool_shape(n, h, w, c));
    TRY(check_channels(c, x_ldc, dtype, "x"));
    TRY(check_channels(c, y_ldc, dtype, "y"));
    TRY(check_ptr(x, "x"));
    TRY(check_ptr(y, "y"));
    if (x_bn) TRY(check_bn(x_bn, "x_bn", true, false));
    if (y_bn) TRY(check_bn(y_bn, "y_bn", false, true));
    TRY(check_ws(ws, ws_bytes, y_bn ? pool_ws(n, h, w, c) : 0));
    MaxPoolParams p;
    memset(&p, 0, sizeof p);
    p.n = n; p.h = h; p.w = w; p.c = c;
    p.ho = (h - 1) / 2 + 1; p.wo = (w - 1) / 2 + 1;
    const int es = esize(dtype);
    const int64_t m = (int64_t)n * h * w, m_out = (int64_t)n * p.ho * p.wo;
    if (overlap(view_range(y, m_out, c, y_ldc, es), view_range(x, m, c, x_ldc, es)))
        return fail(BNR_ERR_ALIAS, "y overlaps x");
    p.x = x; p.x_ldc = x_ldc; p.y = y; p.y_ldc = y_ldc;
    if (x_bn) {
        const Centred cx = centred(x_bn, dt_of(dtype));
        p.gamma = x_bn->gamma; p.beta = x_bn->beta; p.mean = cx.mean; p.rstd = x_bn->rstd; p.ctr = cx.ctr;
    }
    p.part = (float *)ws;
    p.shift = y_bn ? y_bn->shift : nullptr;
    hipStream_t st = (hipStream_t)stream;
    const int dt = dt_of(dtype);
    TRY_HIP(launch_maxpool_fwd(dt, p, x_bn != nullptr, y_bn != nullptr, st), "max pooling");
    if (y_bn) {
        const int64_t R = (int64_t)ceil_div(m_out, ceil_div(m_out, maxpool_fwd_rows(dt, m_out, c)));
        const SplitTerms ft = fwd_terms(y_bn, true);
        TRY_HIP(launch_stats_finalize(p.part, R, c, m_out, FIN_MVF, y_bn->eps, y_bn->mean, y_bn->var, y_bn->rstd,
                                      nullptr, nullptr, (char *)ws + align_up((size_t)pool_ws(n, h, w, c) -
                                                                               align_up(stats_red_bytes(c))),
                                      st, &ft),
                "stats combine");
    }
    return ok();
}

bnr_status bnr_maxpool_bn_bwd(int32_t n, int32_t h, int32_t w, int32_t c, bnr_dtype dtype, const void *x,
                              int32_t x_ldc, const bnr_bn *x_bn, const void *gy, int32_t gy_ldc, void *dy,
                              float *dgamma, float *dbeta, void *ws, size_t ws_bytes, void *stream)
{
    TRY(check_dtype(dtype));
    TRY(check_pool_shape(n, h, w, c));
    TRY(check_channels(c, x_ldc, dtype, "x"));
    TRY(check_channels(c, gy_ldc, dtype, "gy"));
    TRY(check_ptr(x, "x"));
    TRY(check_ptr(gy, "gy"));
    TRY(check_ptr(dy, "dy"));
    const int vec = vec_of(dtype), cvec = c / vec;
    const int wo = (w - 1) / 2 + 1, ho = (h - 1) / 2 + 1;
    if (c > kMaxPoolMaxC || (cvec & (cvec - 1)))
        return fail(BNR_ERR_UNSUPPORTED, "max-pooling backward: %d channels (a power-of-two number of vectors, <= %d)",
                    c, kMaxPoolMaxC);
    if (wo > kMaxPoolMaxWo) return fail(BNR_ERR_UNSUPPORTED, "max-pooling backward: width %d too large", w);
    if (x_bn) {
        TRY(check_bn(x_bn, "x_bn", true, false));
        TRY(check_fptr(dgamma, "dgamma"));
        TRY(check_fptr(dbeta, "dbeta"));
    }
    TRY(check_ws(ws, ws_bytes, x_bn ? pool_ws(n, h, w, c) : 0));
    const int es = esize(dtype);
    const int64_t m = (int64_t)n * h * w, m_out = (int64_t)n * ho * wo;
    const Range rd = view_range(dy, m, c, c, es);
    if (overlap(rd, view_range(x, m, c, x_ldc, es))) return fail(BNR_ERR_ALIAS, "dy overlaps x");
    if (overlap(rd, view_range(gy, m_out, c, gy_ldc, es))) return fail(BNR_ERR_ALIAS, "dy overlaps gy");
    MaxPoolParams p;
    memset(&p, 0, sizeof p);
    p.n = n; p.h = h; p.w = w; p.c = c; p.ho = ho; p.wo = wo;
    p.x = x; p.x_ldc = x_ldc; p.g = gy; p.g_ldc = gy_ldc; p.y = dy; p.y_ldc = c;
    if (x_bn) {
        const Centred cx = centred(x_bn, dt_of(dtype));
        p.gamma = x_bn->gamma; p.beta = x_bn->beta; p.mean = cx.mean; p.rstd = x_bn->rstd; p.ctr = cx.ctr;
    }
    p.part = (float *)ws;
    hipStream_t st = (hipStream_t)stream;
    TRY_HIP(launch_maxpool_bwd(dt_of(dtype), p, x_bn != nullptr, st), "max-pooling backward");
    if (x_bn) {
        const size_t red_off = pool_ws(n, h, w, c) - align_up(stats_red_bytes(c));
        TRY_HIP(launch_stats_finalize(p.part, maxpool_bwd_groups(n, h), c, m, FIN_BWD, 0.f, nullptr, nullptr, nullptr,
                                      dbeta, dgamma, (char *)ws + red_off, st),
                "backward sums combine");
    }
    return ok();
}

size_t bnr_head_workspace_size(int32_t n, int32_t h, int32_t w, int32_t c)
{
    if (n <= 0 || h <= 0 || w <= 0 || c <= 0) return 0;
    return head_ws(n, h, w, c);
}

bnr_status bnr_head_fwd(int32_t n, int32_t h, int32_t w, int32_t c, int32_t classes, bnr_dtype dtype, const void *x,
                        int32_t x_ldc, const bnr_bn *x_bn, const void *wfc, const float *bfc, const int32_t *labels,
                        float *f, float *logits, float *dlogits, float *loss, void *stream)
{
    TRY(check_head(n, h, w, c, classes, dtype, x, x_ldc, x_bn, wfc));
    TRY(check_fptr(bfc, "bfc"));
    if (!labels) return fail(BNR_ERR_NULL, "labels is NULL");
    TRY(check_fptr(f, "f"));
    TRY(check_fptr(logits, "logits"));
    TRY(check_fptr(dlogits, "dlogits"));
    TRY(check_fptr(loss, "loss"));
    HeadParams p;
    head_params(p, dt_of(dtype), n, h, w, c, classes, x, x_ldc, x_bn, wfc);
    p.bfc = bfc; p.labels = labels; p.f = f; p.logits = logits; p.dlogits = dlogits; p.loss = loss;
    TRY_HIP(launch_head_fwd(dt_of(dtype), p, (hipStream_t)stream), "classifier head");
    return ok();
}

bnr_status bnr_head_bwd(int32_t n, int32_t h, int32_t w, int32_t c, int32_t classes, bnr_dtype dtype, const void *x,
                        int32_t x_ldc, const bnr_bn *x_bn, const void *wfc, const float *f, const float *dlogits,
                        float *df, float *dwfc, float *dbfc, float *dgamma, float *dbeta, void *gx, int32_t gx_ldc,
                        float *alpha, float *betap, void *ws, size_t ws_bytes, void *stream)
{
    TRY(check_head(n, h, w, c, classes, dtype, x, x_ldc, x_bn, wfc));
    TRY(check_fptr(f, "f"));
    TRY(check_fptr(dlogits, "dlogits"));
    TRY(check_fptr(df, "df"));
    TRY(check_fptr(dwfc, "dwfc"));
    TRY(check_fptr(dbfc, "dbfc"));
    TRY(check_fptr(dgamma, "dgamma"));
    TRY(check_fptr(dbeta, "dbeta"));
    TRY(check_ptr(gx, "gx"));
    TRY(check_channels(c, gx_ldc, dtype, "gx"));
    const bool split = alpha || betap;
    if (split) {
        TRY(check_fptr(alpha, "alpha"));
        TRY(check_fptr(betap, "betap"));
    }
    TRY(check_ws(ws, ws_bytes, head_ws(n, h, w, c)));
    const int es = esize(dtype);
    const int64_t m = (int64_t)n * h * w;
    if (overlap(view_range(gx, m, c, gx_ldc, es), view_range(x, m, c, x_ldc, es)))
        return fail(BNR_ERR_ALIAS, "gx overlaps x");
    HeadParams p;
    head_params(p, dt_of(dtype), n, h, w, c, classes, x, x_ldc, x_bn, wfc);
    p.f = const_cast<float *>(f);
    p.dlogits = const_cast<float *>(dlogits);
    p.df = df; p.dwfc = dwfc; p.dbfc = dbfc;
    p.gx = gx; p.gx_ldc = gx_ldc;
    p.dgamma = dgamma; p.dbeta = dbeta;
    p.part = (float *)ws;
    const int dt = dt_of(dtype);
    hipStream_t st = (hipStream_t)stream;
    const int64_t R = ceil_div(m, ceil_div(m, head_rows(dt, m, c)));
    void *red = (char *)ws + (head_ws(n, h, w, c) - align_up(stats_red_bytes(c)));
    TRY_HIP(launch_head_bwd_fc(dt, p, st), "classifier head backward");
    if (split) {
        TRY_HIP(launch_head_bn_bwd(dt, p, HB_SPLIT, st), "head BN backward");
        SplitTerms sp{x_bn->gamma, x_bn->rstd, alpha, betap, 0};
        TRY_HIP(launch_stats_finalize(p.part, R, c, m, FIN_BWD, 0.f, nullptr, nullptr, nullptr, dbeta, dgamma, red, st,
                                      &sp),
                "backward sums combine");
    } else {
        TRY_HIP(launch_head_bn_bwd(dt, p, HB_SUMS, st), "head BN backward sums");
        TRY_HIP(launch_stats_finalize(p.part, R, c, m, FIN_BWD, 0.f, nullptr, nullptr, nullptr, dbeta, dgamma, red, st),
                "backward sums combine");
        TRY_HIP(launch_head_bn_bwd(dt, p, HB_DX, st), "head BN input gradient");
    }
    return ok();
}

}  // extern "C"
