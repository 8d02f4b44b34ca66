// conv1x1.hip -- persistent 1x1 CONV (forward and data gradient) on the
// gfx950 matrix cores with the BN fission/fusion prologues and epilogues.
//
// One workgroup per CU (512 threads, 8 waves) keeps the whole weight matrix
// in LDS -- read once from its [c_in][c_out] layout, transposed on load for
// the forward GEMM -- and walks 128-pixel tiles t, t+G, t+2G, ... while every
// workgroup of the grid G has one; the rows left over (fewer than G tiles)
// are split evenly, one short tile per workgroup, so no workgroup runs a
// whole extra tile while the others idle.  For each
// tile the A rows held in registers are transformed by the prologue and
// stored to LDS; the loads of the next tile (and the epilogue operand of this
// tile) are issued before the matrix-core work, so HBM streams while the
// MFMAs run.  The epilogue stages the output tile through LDS so every global
// access is a 16-byte vector of one pixel row, and keeps per-channel
// statistics in registers across all tiles of the workgroup: one partial row
// per workgroup for the float64 combine.
//
// Prologue / epilogue modes are those of conv_rows.hip (PRO_BNRELU, PRO_RELU,
// PRO_BNGRAD, PRO_POOLUP; EPI_STORE, EPI_STATS, EPI_BNBWD, EPI_RELUMASK).
#include "common.hpp"
#include "kernels.hpp"
#include "mfma.hpp"
#include "tiles.hpp"
#include "trace.hpp"

namespace bnr {

constexpr int kP1Threads = 512;
constexpr int kP1BM = 128;     // largest tile height (rows = pixels)
constexpr int kP1NV = 8;       // 16-byte vectors per thread for a tile operand

// Output columns in ncg groups of ncol (the last one may be shorter), each
// computed by gcw workgroups; ncg > 1 only for widths past 256 (the data
// gradient of a wide concatenation), one group per 256 columns at most.
struct P1Geom {
    int KP, NP, lda, ldw, ldc;
    int ncg, ncol, gcw;
    size_t region, lds;
};

// fine: the output columns rounded up to a multiple of 32 (the data gradients
// with the BN-backward epilogue, whose widths are concatenation prefixes:
// 96, 160, 192, 224 channels); otherwise to 32, 64, 128 or 256.
static P1Geom p1_geom(int K, int N, bool fine = false)
{
    P1Geom g;
    g.KP = (K + 31) / 32 * 32;
    g.NP = fine ? (N + 31) / 32 * 32 : (N <= 32 ? 32 : (N <= 64 ? 64 : (N <= 128 ? 128 : 256)));
    g.ncg = 1; g.ncol = N; g.gcw = 1;
    g.lda = g.KP + 8;
    g.ldw = g.KP + 8;
    g.ldc = g.NP + 8;
    const size_t a = (size_t)kP1BM * g.lda, c = (size_t)kP1BM * g.ldc;
    const size_t red = (size_t)2 * (kP1Threads / (g.NP / 8)) * g.NP * sizeof(float) / 2;
    g.region = a > c ? (a > red ? a : red) : (c > red ? c : red);
    g.lds = ((size_t)g.NP * g.ldw + g.region) * 2 + (size_t)(3 * g.KP + 4 * g.NP) * sizeof(float);
    return g;
}

// NVA: upper bound of 16-byte A vectors per thread and tile (compile time, so
// the operand registers stay in VGPRs).  The epilogue kind EK and whether the
// prologue reads a second operand (PRO_BNGRAD) are compile-time as well, so
// the epilogue is straight-line code and the compiler can keep the next
// tile's loads in flight while it waits for the epilogue operand.
// PC: the prologue, compile-time where it pays: PC_BNGRAD (the deferred
// BN input gradient, which reads a second operand), PC_BNRELU (the forward
// BN+ReLU with the statistics epilogue), PC_BNRELU_POOL (BN+ReLU and the 2x2
// average of each window: a tile row loads four input pixels), PC_BNADD (the
// residual block's BN + identity + ReLU: a second operand, and the result is
// stored as a side output), PC_BNRELU_SAVE (BN+ReLU whose result z is also
// stored as a side output: the materialised O2' sweep), PC_RUNTIME (PRO_NONE /
// PRO_BNRELU / PRO_RELU / PRO_POOLUP chosen at run time).
// The BN-backward epilogues read z instead of x when p.e_zsrc is set (see
// the epilogue parameters below).
enum { PC_RUNTIME = 0, PC_BNGRAD = 1, PC_BNRELU = 2, PC_BNRELU_POOL = 3, PC_BNADD = 4, PC_BNRELU_SAVE = 5 };

template <int CBW, int NVA, int EK, int PC, int BM>
__global__ __launch_bounds__(kP1Threads) void k_conv1x1(RowsParams p, P1Geom g)
{
    constexpr bool BNADD = PC == PC_BNADD;
    constexpr bool SAVE = PC == PC_BNRELU_SAVE;
    constexpr bool SIDE = BNADD || SAVE;                  // the transformed A rows are also stored
    constexpr bool BNG = PC == PC_BNGRAD;
    constexpr bool TWO = BNG || BNADD;                     // the prologue reads a second operand
    constexpr bool POOLF = PC == PC_BNRELU_POOL;          // rows are 2x2 windows of the input
    constexpr int PF = POOLF ? 4 : 1;                      // input pixels per A row
    const int pro = PC == PC_BNRELU || POOLF || SIDE ? PRO_BNRELU : (PC == PC_BNGRAD ? PRO_BNGRAD : p.pro);
    using T = bf16_t;
    using M = Mfma<T>;
    constexpr int VEC = 8;
    constexpr int RSTEP_C = kP1Threads / (32 * CBW / VEC);     // epilogue rows per pass
    constexpr int RPT = (BM + RSTEP_C - 1) / RSTEP_C;            // epilogue rows per thread
    constexpr int RB = BM / 64;                                  // 16-row MFMA blocks per wave
    constexpr bool BNBWD = EK == EK_BNBWD || EK == EK_BNBWD_SC || EK == EK_BNBWD_SCACC;
    constexpr bool READS = EK == EK_STORE_ACC || EK == EK_RELUMASK || BNBWD;
    constexpr int NVB = TWO ? NVA : 1, NVX = READS ? RPT : 1, NVD = EK == EK_BNBWD_SCACC ? RPT : 1;
    extern __shared__ __align__(16) unsigned char smem[];
    T *Ws = reinterpret_cast<T *>(smem);
    T *As = Ws + (size_t)g.NP * g.ldw;
    T *Cs = As;                                           // output staging reuses the A tile
    float *coef = reinterpret_cast<float *>(As + g.region);
    float *epi = coef + 3 * g.KP;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;              // 4 x 2 waves: 16 RB rows x NP/2 columns each
    // column group cg: this workgroup's output columns [col0, col0 + N) of NT
    const int cg = (int)blockIdx.x / g.gcw;
    const int col0 = cg * g.ncol, NT = p.N;
    const int N = NT - col0 < g.ncol ? NT - col0 : g.ncol;
    const int K = p.K, KP = g.KP, NP = g.NP;
    const int m = (int)p.m;                               // launcher: m < 2^30
    const int H = p.h, W = p.w;
    const T *wsrc = reinterpret_cast<const T *>(p.wraw);
    const int a_ldc = (int)p.a_ldc, a2_ldc = (int)p.a2_ldc, y_ldc = (int)p.y_ldc, ex_ldc = (int)p.ex_ldc;
    const bool pool = !POOLF && pro == PRO_POOLUP;
    // operand views as raw buffers (launcher guarantees each spans < 2^31 bytes)
    const int64_t arows = pool ? (int64_t)m / 4 : (POOLF ? (int64_t)m * 4 : m);
    const __amdgpu_buffer_rsrc_t abuf = buf_view(p.a, (uint32_t)(((arows - 1) * a_ldc + K) * 2));
    const __amdgpu_buffer_rsrc_t a2buf = buf_view(TWO ? p.a2 : p.a, TWO ? (uint32_t)(((int64_t)(m - 1) * a2_ldc + K) * 2) : 0u);
    const int side_ldc = (int)p.side_ldc;
    const __amdgpu_buffer_rsrc_t sbuf = buf_view(SIDE ? p.side : p.a,
                                                 SIDE ? (uint32_t)(((int64_t)(m - 1) * side_ldc + K) * 2) : 0u);
    const T *ycol = reinterpret_cast<const T *>(p.y) + col0;
    const __amdgpu_buffer_rsrc_t ybuf = buf_view(ycol, (uint32_t)(((int64_t)(m - 1) * y_ldc + N) * 2));
    const __amdgpu_buffer_rsrc_t xbuf = buf_view(p.ex ? reinterpret_cast<const T *>(p.ex) + col0 : ycol,
                                                 p.ex ? (uint32_t)(((int64_t)(m - 1) * ex_ldc + N) * 2) : 0u);
    const int ex2_ldc = (int)p.ex2_ldc;

    // ---- per-channel parameters, loaded first so their round trip overlaps
    // the weights' (KP, NP <= 256 < kP1Threads: thread c holds channel c)
    //   BNRELU: z = max(x * c0 + c1, 0) with c0 = gamma*rstd, c1 = beta - mean*gamma*rstd
    //   BNGRAD: d = c0 * dy + c1 * x + c2  (the deferred BN input gradient: deferred_coef_of)
    float q0 = 0.f, q1 = 0.f, q2 = 0.f, q3 = 0.f, q4 = 0.f;
    if (tid < K && pro == PRO_BNRELU) {
        q0 = p.p_gamma[tid]; q1 = p.p_beta[tid]; q2 = p.p_mean[tid]; q3 = p.p_rstd[tid];
    } else if (tid < K && pro == PRO_BNGRAD) {
        q1 = p.p_mean[tid]; q2 = p.p_rstd[tid];
        if (p.p_split) { q0 = p.p_alpha[tid]; q3 = p.p_betap[tid]; }
        else { q0 = p.p_gamma[tid]; q3 = p.p_dgamma[tid]; q4 = p.p_dbeta[tid]; }
    }
    float ep0 = 0.f, ep1 = 1.f, ep2 = 0.f, ep3 = 0.f;
    if (tid < N && BNBWD) {
        ep0 = p.e_mean[col0 + tid]; ep1 = p.e_rstd[col0 + tid]; ep2 = p.e_gamma[col0 + tid]; ep3 = p.e_beta[col0 + tid];
    }
    if (tid < N && EK == EK_STATS && p.e_shift) ep0 = p.e_shift[col0 + tid];     // statistics of y - shift

    // ---- weights -> LDS as Ws[n][k] (zero outside K x N), in batches of
    // kWB vectors per thread whose loads are all in flight before any write ----
    if (!p.wtrans) {
        // forward W[k][n] -> Ws[n][k]: an item is four consecutive k of one
        // 8-column group (four 16-byte loads), written as one 8-byte word per
        // column (a quarter of the LDS writes of single elements)
        constexpr int kWB = 8, kIB = kWB / 4;
        const __amdgpu_buffer_rsrc_t wbuf = buf_view(wsrc, (uint32_t)(K * NT * 2));
        const int KQ = KP / 4, items = KQ * (NP / VEC);
        for (int base = 0; base < items; base += kIB * kP1Threads) {
            vec16 v[kWB];
            #pragma unroll
            for (int u = 0; u < kWB; u++) {
                if (base + (u >> 2) * kP1Threads >= items) break;   // (uniform: no empty loads issued)
                const int it = base + (u >> 2) * kP1Threads + tid;
                const int n0 = (it / KQ) * VEC, k = (it % KQ) * 4 + (u & 3);
                const int off = it < items && k < K && n0 < N ? (k * NT + col0 + n0) * 2 : (int)kBufOff;
                v[u] = bld16(wbuf, (uint32_t)off);
            }
            #pragma unroll
            for (int ui = 0; ui < kIB; ui++) {
                const int it = base + ui * kP1Threads + tid;
                if (base + ui * kP1Threads >= items) break;
                if (it < items) {
                    const int n0 = (it / KQ) * VEC, k0 = (it % KQ) * 4;
                    #pragma unroll
                    for (int e = 0; e < VEC; e++) {
                        uint32_t h[4];
                        #pragma unroll
                        for (int q = 0; q < 4; q++)
                            h[q] = (e & 1) ? (v[ui * 4 + q].u[e >> 1] >> 16) : (v[ui * 4 + q].u[e >> 1] & 0xffffu);
                        *reinterpret_cast<uint2 *>(Ws + (n0 + e) * g.ldw + k0) =
                            make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
                    }
                }
            }
        }
    } else {
        // data gradient: W[n][k] (n = c_in, k = c_out), rows of k copied straight
        constexpr int kWB = 8;
        const __amdgpu_buffer_rsrc_t wbuf = buf_view(wsrc, (uint32_t)(K * NT * 2));
        const int total = KP * NP / VEC;
        for (int base = 0; base < total; base += kWB * kP1Threads) {
            vec16 v[kWB];
            #pragma unroll
            for (int u = 0; u < kWB; u++) {
                if (base + u * kP1Threads >= total) break;   // (uniform: no empty loads issued)
                const int i = base + u * kP1Threads + tid;
                const int n = i / (KP / VEC), k0 = (i % (KP / VEC)) * VEC;
                const int off = i < total && n < N && k0 < K ? ((col0 + n) * K + k0) * 2 : (int)kBufOff;
                v[u] = bld16(wbuf, (uint32_t)off);
            }
            #pragma unroll
            for (int u = 0; u < kWB; u++) {
                const int i = base + u * kP1Threads + tid;
                if (i >= total) break;
                const int n = i / (KP / VEC), k0 = (i % (KP / VEC)) * VEC;
                *reinterpret_cast<vec16 *>(Ws + n * g.ldw + k0) = v[u];
            }
        }
    }
    // ---- per-channel prologue / epilogue parameters -> LDS ----
    if (tid < KP) {
        float c0 = 0.f, c1 = 0.f, c2 = 0.f;
        if (tid < K && pro == PRO_BNRELU) bn_coef(q0, q1, q2, q3, c0, c1);
        else if (tid < K && pro == PRO_BNGRAD) deferred_coef_of(p.p_split, 1.0f / (float)m, q0, q1, q2, q3, q4, c0, c1, c2);
        coef[tid] = c0; coef[KP + tid] = c1; coef[2 * KP + tid] = c2;
    }
    if (tid < NP) { epi[tid] = ep0; epi[NP + tid] = ep1; epi[2 * NP + tid] = ep2; epi[3 * NP + tid] = ep3; }

    // ---- tile operand registers ----
    // A slot j of this thread: channel vector av of row ar0 + j RPS, with
    // VPR vectors per row and RPS = kP1Threads / VPR rows per step (the
    // launcher checks that NVA slots cover a tile).  Consecutive lanes read
    // consecutive 16-byte vectors of one pixel row (whole rows per wave), and
    // a thread's channels are the same in every slot and every tile, so its
    // prologue coefficients are read from LDS once per launch, not per tile.
    const int VPR = KP / VEC;                          // A vectors per row
    const int RPS = kP1Threads / VPR;
    const int av = tid % VPR, ar0 = tid / VPR;
    int sr[NVA], sc[NVA];
    bool sv[NVA];
    #pragma unroll
    for (int j = 0; j < NVA; j++) {
        sr[j] = ar0 + j * RPS;
        sc[j] = av * VEC;
        sv[j] = ar0 < RPS && sr[j] < BM;
    }
    float kc0[VEC], kc1[VEC], kc2[VEC];                // its prologue coefficients (set below)
    vec16 ra[NVA * PF], rb[NVB];
    // the wave-uniform mode switches sit outside the slot loops, so each
    // mode's slots are straight-line code
    auto load_a = [&](int p0, int lim) __attribute__((always_inline)) {
        if (POOLF) {                    // row q = window (img, y, x) of the (H/2) x (W/2) grid
            const int ho = H / 2, wo = W / 2;
            #pragma unroll
            for (int j = 0; j < NVA; j++) {
                const int q = p0 + sr[j], c = sc[j];
                const bool ok = sv[j] && c < K && q < lim;
                const int img = q / (ho * wo);
                const int rem = q - img * ho * wo;
                const int y = rem / wo, x = rem - y * wo;
                const int p00 = (img * H + 2 * y) * W + 2 * x;
                #pragma unroll
                for (int f = 0; f < 4; f++) {
                    const int pp = p00 + (f >> 1) * W + (f & 1);
                    ra[j * PF + f] = bld16(abuf, ok ? (uint32_t)(pp * a_ldc + c) * 2u : kBufOff);
                }
            }
        } else if (!BNG && pool) {      // (the deferred-gradient variants never read a pooled gradient)
            #pragma unroll
            for (int j = 0; j < NVA; j++) {
                const int pp = p0 + sr[j], c = sc[j];
                const bool ok = sv[j] && c < K && pp < lim;
                const int img = pp / (H * W);
                const int rem = pp - img * H * W;
                const int y = rem / W, x = rem - y * W;
                const int q = (img * (H / 2) + y / 2) * (W / 2) + x / 2;
                ra[j] = bld16(abuf, ok ? (uint32_t)(q * a_ldc + c) * 2u : kBufOff);
            }
        } else {
            #pragma unroll
            for (int j = 0; j < NVA; j++) {
                const int pp = p0 + sr[j], c = sc[j];
                const bool ok = sv[j] && c < K && pp < lim;
                ra[j] = bld16(abuf, ok ? (uint32_t)(pp * a_ldc + c) * 2u : kBufOff);
                if (TWO) rb[j < NVB ? j : 0] = bld16(a2buf, ok ? (uint32_t)(pp * a2_ldc + c) * 2u : kBufOff);
            }
        }
    };
    // Prologue transforms.  A 1x1 output row depends on its own input row
    // only, so rows past the end need no masking (their outputs are never
    // stored or counted); channels past K read zeros and have zero
    // coefficients and zero weights.
    auto store_a = [&](int p0, int lim) __attribute__((always_inline)) {
        auto put = [&](int j, const vec16 &v) __attribute__((always_inline)) {
            if (sv[j]) *reinterpret_cast<vec16 *>(As + sr[j] * g.lda + sc[j]) = v;
        };
        if (BNADD) {                                      // r = max(y c0 + c1 + identity, 0), also stored
            #pragma unroll
            for (int j = 0; j < NVA; j++) {
                float f[VEC], id[VEC];
                Elem<T>::unpack(ra[j], f);
                Elem<T>::unpack(rb[j < NVB ? j : 0], id);
                #pragma unroll
                for (int e = 0; e < VEC; e++) f[e] = __builtin_fmaxf(bn_lin(f[e], kc0[e], kc1[e]) + id[e], 0.f);
                const vec16 v = Elem<T>::pack(f);
                put(j, v);
                const int pp = p0 + sr[j];
                bst16(sbuf, sv[j] && sc[j] < K && pp < lim ? (uint32_t)(pp * side_ldc + sc[j]) * 2u : kBufOff, v);
            }
        } else if (BNG) {                                        // PRO_BNGRAD: d = c0 dy + c1 x + c2
            #pragma unroll
            for (int j = 0; j < NVA; j++) {
                float f[VEC], x[VEC];
                Elem<T>::unpack(ra[j], f);
                Elem<T>::unpack(rb[j < NVB ? j : 0], x);
                #pragma unroll
                for (int e = 0; e < VEC; e++) f[e] = __builtin_fmaf(kc0[e], f[e], __builtin_fmaf(kc1[e], x[e], kc2[e]));
                put(j, Elem<T>::pack(f));
            }
        } else if (POOLF) {                               // z = mean over the window of max(x c0 + c1, 0)
            #pragma unroll
            for (int j = 0; j < NVA; j++) {
                float acc[VEC];
                #pragma unroll
                for (int e = 0; e < VEC; e++) acc[e] = 0.f;
                #pragma unroll
                for (int f4 = 0; f4 < PF; f4++) {
                    float f[VEC];
                    Elem<T>::unpack(ra[j * PF + f4], f);
                    #pragma unroll
                    for (int e = 0; e < VEC; e++) acc[e] += __builtin_fmaxf(bn_lin(f[e], kc0[e], kc1[e]), 0.f);
                }
                #pragma unroll
                for (int e = 0; e < VEC; e++) acc[e] *= 0.25f;
                put(j, Elem<T>::pack(acc));
            }
        } else if (pro == PRO_BNRELU) {                   // z = max(x c0 + c1, 0)   (SAVE: also stored)
            #pragma unroll
            for (int j = 0; j < NVA; j++) {
                float f[VEC];
                Elem<T>::unpack(ra[j], f);
                #pragma unroll
                for (int e = 0; e < VEC; e++) {
                    const float t = bn_lin(f[e], kc0[e], kc1[e]);
                    f[e] = t > 0.f ? t : 0.f;
                }
                const vec16 v = Elem<T>::pack(f);
                put(j, v);
                if (SAVE) {
                    const int pp = p0 + sr[j];
                    bst16(sbuf, sv[j] && sc[j] < K && pp < lim ? (uint32_t)(pp * side_ldc + sc[j]) * 2u : kBufOff, v);
                }
            }
        } else if (pro == PRO_RELU) {
            #pragma unroll
            for (int j = 0; j < NVA; j++) {
                float f[VEC];
                Elem<T>::unpack(ra[j], f);
                #pragma unroll
                for (int e = 0; e < VEC; e++) f[e] = f[e] > 0.f ? f[e] : 0.f;
                put(j, Elem<T>::pack(f));
            }
        } else if (!BNG && pool) {                        // PRO_POOLUP: g[p/2] / 4
            #pragma unroll
            for (int j = 0; j < NVA; j++) {
                float f[VEC];
                Elem<T>::unpack(ra[j], f);
                #pragma unroll
                for (int e = 0; e < VEC; e++) f[e] *= 0.25f;
                put(j, Elem<T>::pack(f));
            }
        } else {
            #pragma unroll
            for (int j = 0; j < NVA; j++) put(j, ra[j]);
        }
    };

    // ---- epilogue mapping: thread = one channel vector of rows r0, r0+RSTEP, ...
    // (a width that does not divide the workgroup leaves its last threads idle) ----
    const int VPRO = NP / VEC, RSTEP = RSTEP_C;
    const int v = tid % VPRO, r0 = tid / VPRO;
    const int n = v * VEC;
    const bool act = r0 < RSTEP;
    const bool col_ok = act && n < N;
    vec16 rx[NVX], rd[NVD];
    float s1[VEC], s2[VEC];
    #pragma unroll
    for (int e = 0; e < VEC; e++) { s1[e] = 0.f; s2[e] = 0.f; }
    T *yout = reinterpret_cast<T *>(p.y) + col0;

    __syncthreads();
    // this thread's prologue channels are fixed too: their coefficients in registers
    if (pro == PRO_BNRELU || pro == PRO_BNGRAD) {
        lds_f8(coef + av * VEC, kc0);
        lds_f8(coef + KP + av * VEC, kc1);
        if (pro == PRO_BNGRAD) lds_f8(coef + 2 * KP + av * VEC, kc2);
        else
            #pragma unroll
            for (int e = 0; e < VEC; e++) kc2[e] = 0.f;
    } else {
        #pragma unroll
        for (int e = 0; e < VEC; e++) { kc0[e] = 0.f; kc1[e] = 0.f; kc2[e] = 0.f; }
    }
    // this thread's epilogue channels are fixed: keep their BN parameters in registers
    float eM[VEC], eR[VEC], eG[VEC], eB[VEC], eC0[VEC], eC1[VEC], eS[VEC];
    #pragma unroll
    for (int e = 0; e < VEC; e++) {
        eM[e] = epi[n + e]; eR[e] = epi[NP + n + e]; eG[e] = epi[2 * NP + n + e]; eB[e] = epi[3 * NP + n + e];
        bn_coef(eG[e], eB[e], eM[e], eR[e], eC0[e], eC1[e]);     // the forward prologue's y = x c0 + c1
        eS[e] = eC0[e];                                           // summed-gradient scale gamma rstd
    }
    // e_zsrc: the BN-backward operand is the stored z = relu(y) (the O2' sweep):
    // mask [z > 0] (as fma(z, 1, 0) > 0) and xhat = (z - beta) / gamma where the
    // mask passes; a thread whose channel vector holds a gamma = 0 channel
    // (xhat not recoverable from z) reads x (ex2) with the usual parameters.
    const bool zsrc = BNBWD && p.e_zsrc;
    bool zs = zsrc && col_ok;
    #pragma unroll
    for (int e = 0; e < VEC; e++) zs = zs && eG[e] != 0.f;
    if (zs)
        #pragma unroll
        for (int e = 0; e < VEC; e++) { eM[e] = eB[e]; eR[e] = 1.0f / eG[e]; eC0[e] = 1.f; eC1[e] = 0.f; }
    // (the z / x source of this thread's channel vector as a plain pointer:
    // the choice is per lane, so one load replaces two raw-buffer loads merged
    // after both arrive)
    const T *zsrc_col = reinterpret_cast<const T *>(zs ? p.ex : (p.ex2 ? p.ex2 : p.ex)) + col0 + (col_ok ? n : 0);
    const int zsrc_ldc = zs ? ex_ldc : ex2_ldc;
    auto load_epi = [&](int p0, int lim) __attribute__((always_inline)) {
        if (!READS) return;
        #pragma unroll
        for (int j = 0; j < NVX; j++) {
            const int r = r0 + j * RSTEP, pp = p0 + r;
            const bool ok = col_ok && r < BM && pp < lim;
            if (EK == EK_STORE_ACC) {
                rx[j] = bld16(ybuf, ok ? (uint32_t)(pp * y_ldc + n) * 2u : kBufOff);
            } else if (BNBWD && zsrc) {   // z, or x for a vector holding a gamma = 0 channel: one load
                // from this thread's source at a clamped row (a row past the tile is not used)
                rx[j] = ldg16(zsrc_col + (int64_t)(ok ? pp : 0) * zsrc_ldc);
            } else {
                rx[j] = bld16(xbuf, ok ? (uint32_t)(pp * ex_ldc + n) * 2u : kBufOff);
            }
            if (EK == EK_BNBWD_SCACC) rd[j < NVD ? j : 0] = bld16(ybuf, ok ? (uint32_t)(pp * y_ldc + n) * 2u : kBufOff);
        }
    };
    // work items: F rounds of whole tiles (item k < F is tile k*G + gi, rows
    // [p0, p0 + BM)), then this workgroup's share [lo, hi) of the R rows left
    const int G = g.gcw, gi = (int)blockIdx.x - cg * g.gcw;
    const int F = m / (G * BM), R = m - F * G * BM;         // R < G*BM <= 2^16, so gi*R fits
    const int lo = F * G * BM + gi * R / G, hi = F * G * BM + (gi + 1) * R / G;
    const int nitems = F + (hi > lo ? 1 : 0);
    auto item = [&](int k, int &p0, int &lim) __attribute__((always_inline)) {
        if (k < F) { p0 = (k * G + gi) * BM; lim = p0 + BM; } else { p0 = lo; lim = hi; }
    };
    if (nitems > 0) { int q0, ql; item(0, q0, ql); load_a(q0, ql); }
    for (int k = 0; k < nitems; k++) {
        int p0, lim;
        item(k, p0, lim);
        // epilogue operand first, before this tile's staging: it then has the
        // staging, the matrix cores and the output staging to arrive, and the
        // staging's wait for this tile's rows (issued earlier) leaves it in
        // flight; the next tile's rows follow it
        load_epi(p0, lim);
        store_a(p0, lim);
        __syncthreads();
        if (k + 1 < nitems) { int q0, ql; item(k + 1, q0, ql); load_a(q0, ql); }
        // ---- matrix cores: 16 RB rows x NP/2 columns per wave ----
        f32x4 acc[RB][CBW];
        #pragma unroll
        for (int ib = 0; ib < RB; ib++)
            #pragma unroll
            for (int cb = 0; cb < CBW; cb++) acc[ib][cb] = f32x4{0.f, 0.f, 0.f, 0.f};
        const T *arow = As + (wm * (16 * RB) + (lane & 15)) * g.lda + (lane >> 4) * M::KPL;
        const T *brow = Ws + (wn * (NP / 2) + (lane & 15)) * g.ldw + (lane >> 4) * M::KPL;
        // (a wave whose 16*RB rows all lie past the end of a short tile skips them)
        for (int k0 = 0; k0 < (wm * 16 * RB < lim - p0 ? KP : 0); k0 += M::KSTEP) {
            typename M::frag a[RB];
            #pragma unroll
            for (int ib = 0; ib < RB; ib++) a[ib] = M::load(arow + ib * 16 * g.lda + k0);
            #pragma unroll
            for (int cb = 0; cb < CBW; cb++) {
                const typename M::frag b = M::load(brow + cb * 16 * g.ldw + k0);
                #pragma unroll
                for (int ib = 0; ib < RB; ib++) M::mma(acc[ib][cb], b, a[ib]);
            }
        }
        __syncthreads();
        // (the weights are the matrix cores' first operand, so a lane holds
        // four consecutive channels of one pixel row: one 8-byte write)
        #pragma unroll
        for (int ib = 0; ib < RB; ib++)
            #pragma unroll
            for (int cb = 0; cb < CBW; cb++) {
                const int row = wm * (16 * RB) + ib * 16 + (lane & 15);
                const int col = wn * (NP / 2) + cb * 16 + (lane >> 4) * 4;
                const uint2 w = make_uint2(pack2bf(acc[ib][cb][0], acc[ib][cb][1]), pack2bf(acc[ib][cb][2], acc[ib][cb][3]));
                *reinterpret_cast<uint2 *>(Cs + row * g.ldc + col) = w;
            }
        __syncthreads();
        // ---- epilogue row pass: all outputs of this thread first (invalid rows
        // contribute zeros), then the stores back to back ----
        vec16 vo[RPT];
        #pragma unroll
        for (int j = 0; j < RPT; j++) {
            const int r = r0 + j * RSTEP;
            const bool ok = col_ok && r < BM && p0 + r < lim;
            const vec16 cv = *reinterpret_cast<const vec16 *>(Cs + (r < BM ? r : 0) * g.ldc + n);
            float f[VEC];
            Elem<T>::unpack(cv, f);
            vo[j] = cv;
            if (EK == EK_STORE_ACC) {
                float old[VEC];
                Elem<T>::unpack(rx[j < NVX ? j : 0], old);
                #pragma unroll
                for (int e = 0; e < VEC; e++) f[e] += old[e];
                vo[j] = Elem<T>::pack(f);
            } else if (EK == EK_STATS) {
                #pragma unroll
                for (int e = 0; e < VEC; e++) {
                    const float fv = ok ? f[e] - eM[e] : 0.f;
                    s1[e] += fv;
                    s2[e] += fv * fv;
                }
            } else if (EK == EK_RELUMASK) {
                float yv[VEC];
                Elem<T>::unpack(rx[j < NVX ? j : 0], yv);
                #pragma unroll
                for (int e = 0; e < VEC; e++) f[e] = yv[e] > 0.f ? f[e] : 0.f;
                vo[j] = Elem<T>::pack(f);
            } else if (BNBWD) {
                float x[VEC], old[VEC];
                Elem<T>::unpack(rx[j < NVX ? j : 0], x);
                if (EK == EK_BNBWD_SCACC) Elem<T>::unpack(rd[j < NVD ? j : 0], old);
                #pragma unroll
                for (int e = 0; e < VEC; e++) {
                    const float xh = (x[e] - eM[e]) * eR[e];
                    const float d = ok && bn_lin(x[e], eC0[e], eC1[e]) > 0.f ? f[e] : 0.f;
                    s1[e] += d;
                    s2[e] += d * xh;
                    if (EK == EK_BNBWD) f[e] = d;
                    else if (EK == EK_BNBWD_SC) f[e] = d * eS[e];
                    else f[e] = __builtin_fmaf(d, eS[e], old[e]);
                }
                vo[j] = Elem<T>::pack(f);
            }
        }
        #pragma unroll
        for (int j = 0; j < RPT; j++) {
            const int r = r0 + j * RSTEP;
            if (col_ok && r < BM && p0 + r < lim) stg16(yout + (int64_t)(p0 + r) * y_ldc + n, vo[j]);
        }
        __syncthreads();
    }

    // ---- per-workgroup statistics partial row ----
    if (EK == EK_STATS || BNBWD) {
        float *red = reinterpret_cast<float *>(As);
        if (act)
            #pragma unroll
            for (int e = 0; e < VEC; e++) {
                red[r0 * NP + n + e] = s1[e];
                red[(RSTEP + r0) * NP + n + e] = s2[e];
            }
        lds_colsum2(red, RSTEP, NP, NP, kP1Threads, tid, p.part + (int64_t)gi * 2 * NT + col0,
                    p.part + (int64_t)gi * 2 * NT + NT + col0, N);
    }
}

// ------------------------------------------------------------- launchers ---
static int device_cus()
{
    static int cus = 0;
    if (!cus) {
        int dev = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
            cus = 256;
    }
    return cus;
}

// Column groups: one up to 256 output columns; the data gradient with the
// BN-backward epilogue (the gradient of a wide concatenation) takes up to
// kP1MaxN columns in the fewest groups of equal width (rounded up to 32, at
// most 256) whose weight columns and staging fit the LDS.  Every group
// re-reads the A rows (K <= 256 channels, small beside the epilogue's three
// N-wide sweeps).
constexpr int kP1MaxN = 2048;
constexpr size_t kP1MaxLds = 150 * 1024;
static int p1_group_cols(int K, int N)
{
    if (N <= 256) return N;
    for (int64_t ncg = ceil_div(N, 256); ncg <= ceil_div(N, 32); ncg++) {
        const int ncol = (int)(ceil_div(ceil_div(N, ncg), 32) * 32);
        if (p1_geom(K, ncol).lds <= kP1MaxLds) return ncol;
    }
    return 32;
}

bool conv1x1_supported(int dtype, int K, int N, int epi)
{
    if (dtype != DT_BF16 || K > 256 || N < 1 || N > kP1MaxN || (N > 256 && epi != EPI_BNBWD)) return false;
    const P1Geom g = p1_geom(K, p1_group_cols(K, N));
    if (g.lds > kP1MaxLds) return false;
    if ((int64_t)kP1BM * (g.KP / 8) > (int64_t)kP1NV * kP1Threads) return false;      // A tile registers
    if (kP1BM / (kP1Threads / (g.NP / 8)) > kP1NV) return false;                       // epilogue registers
    return true;
}

// One workgroup per CU (see run_p1): at most one partial row per CU.
int64_t conv1x1_partial_rows(int64_t m)
{
    const int64_t tiles = ceil_div(m, 64);
    const int64_t g = device_cus();
    return tiles < g ? tiles : g;
}

template <int CBW, int NVA, int EK, int PC, int BM>
static hipError_t run_p1(const RowsParams &p, const P1Geom &g, hipStream_t s, int64_t *rows)
{
    constexpr bool BNG = PC == PC_BNGRAD;
    auto kern = k_conv1x1<CBW, NVA, EK, PC, BM>;
    static bool attr_set = false;
    if (!attr_set) {
        const hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    // one workgroup per CU: a second one (where registers and LDS would allow
    // it) measured no faster and doubles the statistics partial rows
    const int ntiles = (int)ceil_div(p.m, BM);
    const int64_t gmax = device_cus();
    const int64_t per_group = gmax / g.ncg > 1 ? gmax / g.ncg : 1;
    P1Geom gg = g;
    gg.gcw = (int)(ntiles < per_group ? ntiles : per_group);
    // a thread's NVA A slots step over rows kP1Threads / (KP / 8) apart: they must cover a tile
    const int rps = kP1Threads / (g.KP / 8);
    if ((BM + rps - 1) / rps > NVA) return hipErrorInvalidValue;
    const int grid = gg.gcw * g.ncg;
    *rows = gg.gcw;
    const double m = (double)p.m;
    double a = m * p.K;
    if (BNG) a *= 2.0;
    if (PC == PC_BNADD) a *= 3.0;                   // y and the identity read, the result written
    if (PC == PC_BNRELU_SAVE) a *= 2.0;             // x read, z written
    if (p.pro == PRO_POOLUP) a /= 4.0;
    if (PC == PC_BNRELU_POOL) a *= 4.0;             // four input pixels per row
    double out = m * p.N;
    if (EK == EK_STORE_ACC || EK == EK_RELUMASK || EK == EK_BNBWD || EK == EK_BNBWD_SC) out += m * p.N;
    if (EK == EK_BNBWD_SCACC) out += 2.0 * m * p.N;
    TraceScope tr(KC_CONV, KID_CONV_1X1, s, 2.0 * (a + out + (double)p.K * p.N), 2.0 * m * p.K * p.N);
    hipLaunchKernelGGL(kern, dim3(grid), dim3(kP1Threads), g.lds, s, p, gg);
    return hipGetLastError();
}

// Tile height: 128 rows unless the operand registers of the variant would not
// fit the 256 VGPRs a wave has at two waves per SIMD; then 64 rows, which
// halves every per-thread operand array.
template <int CBW, int NVA128, int EK, int PC>
static hipError_t run_p1_bm(const RowsParams &p, const P1Geom &g, hipStream_t s, int64_t *rows)
{
    constexpr bool reads = EK == EK_STORE_ACC || EK == EK_RELUMASK || EK >= EK_BNBWD;
    constexpr bool small = (CBW >= 5 && reads) || (NVA128 == 8 && (PC == PC_BNGRAD || PC == PC_BNADD)) ||
                           PC == PC_BNRELU_POOL;
    // (64-row tiles hold at most four 16-byte A vectors per thread; the
    // pooling prologue loads four pixels for each)
    if constexpr (small) return run_p1<CBW, 4, EK, PC, 64>(p, g, s, rows);
    else return run_p1<CBW, NVA128, EK, PC, 128>(p, g, s, rows);
}

template <int NVA128, int EK, int PC>
static hipError_t run_p1_cbw(const RowsParams &p, const P1Geom &g, hipStream_t s, int64_t *rows)
{
    constexpr bool FINE = EK == EK_BNBWD || EK == EK_BNBWD_SC || EK == EK_BNBWD_SCACC;
    switch (g.NP / 32) {
    case 1: return run_p1_bm<1, NVA128, EK, PC>(p, g, s, rows);
    case 2: return run_p1_bm<2, NVA128, EK, PC>(p, g, s, rows);
    case 4: return run_p1_bm<4, NVA128, EK, PC>(p, g, s, rows);
    case 8: return run_p1_bm<8, NVA128, EK, PC>(p, g, s, rows);
    default: break;
    }
    if constexpr (FINE) {
        switch (g.NP / 32) {
        case 3: return run_p1_bm<3, NVA128, EK, PC>(p, g, s, rows);
        case 5: return run_p1_bm<5, NVA128, EK, PC>(p, g, s, rows);
        case 6: return run_p1_bm<6, NVA128, EK, PC>(p, g, s, rows);
        case 7: return run_p1_bm<7, NVA128, EK, PC>(p, g, s, rows);
        default: break;
        }
    }
    return hipErrorInvalidValue;
}

template <int EK, int PC>
static hipError_t run_p1_nva(const RowsParams &p, const P1Geom &g, hipStream_t s, int64_t *rows)
{
    const int nva = (int)ceil_div((int64_t)kP1BM * (g.KP / 8), kP1Threads);
    if (nva <= 4) return run_p1_cbw<4, EK, PC>(p, g, s, rows);
    return run_p1_cbw<8, EK, PC>(p, g, s, rows);
}

template <int PC>
static hipError_t run_p1_ek(const RowsParams &p, const P1Geom &g, int ek, hipStream_t s, int64_t *rows)
{
    switch (ek) {
    case EK_STORE: return run_p1_nva<EK_STORE, PC>(p, g, s, rows);
    case EK_STORE_ACC: return run_p1_nva<EK_STORE_ACC, PC>(p, g, s, rows);
    case EK_STATS: return run_p1_nva<EK_STATS, PC>(p, g, s, rows);
    case EK_RELUMASK: return run_p1_nva<EK_RELUMASK, PC>(p, g, s, rows);
    case EK_BNBWD_SC: return run_p1_nva<EK_BNBWD_SC, PC>(p, g, s, rows);
    case EK_BNBWD_SCACC: return run_p1_nva<EK_BNBWD_SCACC, PC>(p, g, s, rows);
    default: return run_p1_nva<EK_BNBWD, PC>(p, g, s, rows);
    }
}

hipError_t launch_conv1x1(const RowsParams &p, hipStream_t s, int64_t *rows)
{
    if (!p.a || !p.wraw || !p.y || p.taps != 1 || !conv1x1_supported(p.dtype, p.K, p.N, p.epi)) return hipErrorInvalidValue;
    if (p.pro == PRO_BNRELU && (!p.p_mean || !p.p_gamma || !p.p_rstd || !p.p_beta)) return hipErrorInvalidValue;
    if (p.pro == PRO_BNGRAD && (!p.a2 || !p.p_mean || !p.p_rstd ||
                                (p.p_split ? (!p.p_alpha || !p.p_betap) : (!p.p_gamma || !p.p_dbeta || !p.p_dgamma))))
        return hipErrorInvalidValue;
    if ((p.epi == EPI_STATS || p.epi == EPI_BNBWD) && !p.part) return hipErrorInvalidValue;
    if (p.epi == EPI_BNBWD && (!p.ex || !p.e_mean || !p.e_rstd || !p.e_gamma || !p.e_beta)) return hipErrorInvalidValue;
    if (p.epi == EPI_RELUMASK && !p.ex) return hipErrorInvalidValue;
    if (p.pro == PRO_POOLUP && (p.h % 2 || p.w % 2 || (int64_t)p.n * p.h * p.w != p.m)) return hipErrorInvalidValue;
    const bool poolf = p.pro == PRO_BNRELU_POOL;
    if (poolf && (p.h % 2 || p.w % 2 || (int64_t)p.n * p.h * p.w != 4 * p.m || p.wtrans ||
                  (p.epi != EPI_STORE && p.epi != EPI_STATS) || p.accumulate || !p.p_mean || !p.p_gamma ||
                  !p.p_rstd || !p.p_beta))
        return hipErrorInvalidValue;
    const bool bnadd = p.pro == PRO_BNADDRELU;
    if (bnadd && (!p.a2 || !p.side || p.wtrans || (p.epi != EPI_STORE && p.epi != EPI_STATS) || p.accumulate ||
                  !p.p_mean || !p.p_gamma || !p.p_rstd || !p.p_beta))
        return hipErrorInvalidValue;
    const bool save = p.pro == PRO_BNRELU && p.side;
    if (save && (p.wtrans || (p.epi != EPI_STORE && p.epi != EPI_STATS) || p.accumulate)) return hipErrorInvalidValue;
    if (p.side && !bnadd && !save) return hipErrorInvalidValue;
    if (p.e_zsrc && (p.epi != EPI_BNBWD || !p.ex2)) return hipErrorInvalidValue;
    // 32-bit pixel indices and raw-buffer operand views: every span below 2^31 bytes
    const int64_t lim = (int64_t)1 << 31;
    const int64_t arows = poolf ? 4 * p.m : p.m;
    if ((bnadd || save) && (p.m * p.side_ldc + p.K) * 2 >= lim) return hipErrorInvalidValue;
    if (p.ex2 && (p.m * p.ex2_ldc + p.N) * 2 >= lim) return hipErrorInvalidValue;
    if (p.m < 1 || arows >= (lim >> 1) || (arows * p.a_ldc + p.K) * 2 >= lim || (p.m * p.y_ldc + p.N) * 2 >= lim ||
        (p.a2 && (p.m * p.a2_ldc + p.K) * 2 >= lim) || (p.ex && (p.m * p.ex_ldc + p.N) * 2 >= lim))
        return hipErrorInvalidValue;
    const int ncol = p1_group_cols(p.K, p.N);
    P1Geom g = p1_geom(p.K, ncol, p.epi == EPI_BNBWD);
    g.ncg = (int)ceil_div(p.N, ncol);
    g.ncol = ncol;
    const int ek = epilogue_kind(p.epi, p.accumulate, p.e_scale);
    if (poolf) return ek == EK_STATS ? run_p1_nva<EK_STATS, PC_BNRELU_POOL>(p, g, s, rows)
                                     : run_p1_nva<EK_STORE, PC_BNRELU_POOL>(p, g, s, rows);
    if (bnadd) return ek == EK_STATS ? run_p1_nva<EK_STATS, PC_BNADD>(p, g, s, rows)
                                     : run_p1_nva<EK_STORE, PC_BNADD>(p, g, s, rows);
    if (save) return ek == EK_STATS ? run_p1_nva<EK_STATS, PC_BNRELU_SAVE>(p, g, s, rows)
                                    : run_p1_nva<EK_STORE, PC_BNRELU_SAVE>(p, g, s, rows);
    if (p.pro == PRO_BNGRAD) return run_p1_ek<PC_BNGRAD>(p, g, ek, s, rows);
    if (p.pro == PRO_BNRELU && ek == EK_STATS) return run_p1_nva<EK_STATS, PC_BNRELU>(p, g, s, rows);
    return run_p1_ek<PC_RUNTIME>(p, g, ek, s, rows);
}

}  // namespace bnr
