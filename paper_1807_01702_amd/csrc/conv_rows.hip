// conv_rows.hip -- implicit-GEMM CONV over NHWC pixel rows on the gfx950
// matrix cores, with the BN fission/fusion prologues and epilogues.
//
// GEMM view: M = pixels, N = output channels, K = taps x input channels.
// The same kernel runs the forward CONV and the data gradient (the data
// gradient of a stride-1 zero-padded CONV is a forward CONV of the output
// gradient with the filter taps flipped and c_in/c_out swapped; the weight
// packer produces that operand).
//
// Per workgroup: a BM x BN output tile.  K is consumed in chunks of 32 input
// channels; for each chunk the workgroup stages (a) the A rows of its pixels
// plus, for 3x3, a halo of W+1 pixel rows on each side, already transformed
// by the prologue and rounded to the matrix-core operand type, and (b) the
// packed weights of all taps of the chunk.  Each tap then reads its shifted
// A rows from LDS; taps that leave the image read 0 (zero padding applies to
// the CONV input, i.e. after BN and ReLU).
//
// Prologues (sub-BN2 side, Sec. 3.2):
//   PRO_RELU   : a = max(x, 0)   (ReLU-CONV fusion alone, unfused-BN modes)
//   PRO_BNRELU : a = max(gamma*(x-mean)*rstd + beta, 0); with p.side set, a
//                is also stored there (the materialised O2' sweep; general
//                staging loop, by the first column tile, the tile's own rows)
//   PRO_BNGRAD : a = A dy + B x + C  (deferred BN input gradient from dy and
//                the BN input x; coefficients by deferred_coef)
//   PRO_POOLUP : a = g[n][y/2][x/2] / 4   (2x2 average-pooling gradient)
//   PRO_BNRELU_POOL: row = 2x2 window; a = mean over its four pixels of
//                max(gamma*(x-mean)*rstd + beta, 0)  (1x1 only, general
//                staging loop)
//   PRO_BNADDRELU: a = max(gamma*(x-mean)*rstd + beta + r0, 0), r0 the
//                identity (a2); a is also stored to the side view (1x1 only,
//                general staging loop, by the first column tile)
// Epilogues (sub-BN1 side):
//   EPI_STATS  : store y, per-channel sum(y), sum(y^2) of the stored values
//   EPI_BNBWD  : dy = dz * [gamma*xhat+beta > 0] with xhat from the BN input,
//                store dy (e_scale: store or add gamma*rstd*dy), per-channel
//                sum(dy), sum(dy*xhat); with e_zsrc, ex is the stored
//                z = relu(y): mask [z > 0], xhat = (z - beta)/gamma, and a
//                thread whose channel vector holds a gamma = 0 channel reads
//                x (ex2) with the usual formulas instead
//   EPI_RELUMASK: dy = dz * [y > 0] from a stored y (ReLU-CONV fusion alone)
// float32 data: x - mean in the prologues and the BN-backward epilogue is
// (x - K) - (mean - K) with the BN's centre K (bn_centre), x in PRO_BNGRAD is
// x - K with the coefficients formed from mean - K.
// The epilogue goes through LDS so that every global access is a 16-byte
// vector of one pixel row.
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"
#include "mfma.hpp"
#include "tiles.hpp"
#include "trace.hpp"

namespace bnr {

// BK: input channels per K chunk (kRowsBK, or kRowsBKDirect for the
// specialised bf16 1x1 cases below, whose weights are staged either as rows
// of n ([n][k], pitch ASTR) or as rows of k ([k][n], pitch BN + 8)).
template <typename T, int TAPS, int BM, int BN, int BK = kRowsBK>
struct RowsCfg {
    static constexpr int VEC = Elem<T>::VEC;
    static constexpr int PAD = 16 / (int)sizeof(T);
    static constexpr int ASTR = BK + PAD;                      // staged row stride (elements)
    static constexpr int HALO_MAX = TAPS == 9 ? kRowsMaxW3 + 1 : 0;
    static constexpr int AROWS = BM + 2 * HALO_MAX;
    static constexpr int A_ELEMS = AROWS * ASTR;
    static constexpr int B_ELEMS = TAPS * (BN * ASTR > BK * (BN + 8) ? BN * ASTR : BK * (BN + 8));
    static constexpr int CSTR = BN + PAD;
    static constexpr size_t STAGE_BYTES = (size_t)(A_ELEMS + B_ELEMS) * sizeof(T);
    static constexpr size_t EPI_BYTES = (size_t)BM * CSTR * sizeof(T);
    static constexpr int RSTEP = kThreads / (BN / VEC);
    static constexpr size_t RED_BYTES = 2ull * RSTEP * BN * sizeof(float);
    static constexpr size_t LDS = STAGE_BYTES > EPI_BYTES ? (STAGE_BYTES > RED_BYTES ? STAGE_BYTES : RED_BYTES)
                                                          : (EPI_BYTES > RED_BYTES ? EPI_BYTES : RED_BYTES);
};

// SP: a compile-time case of the pipelined bf16 1x1 path (caller's weights,
// every span below 2^31 bytes), so its chunk loop has no mode branches:
// SP_FWD_BNRELU: forward, BN+ReLU prologue, weights [k][n];
// SP_DGRAD_BNGRAD: data gradient, deferred-gradient prologue, weights [n][k];
// SP_RUNTIME: every mode, chosen at run time.  With one workgroup per CU, as
// in late dense blocks, the mode branches are on the critical path (forward
// about 20% of the launch, data gradient about 6%).
enum { SP_RUNTIME = 0, SP_FWD_BNRELU = 1, SP_DGRAD_BNGRAD = 2 };
// K chunk of the forward case: a wider chunk means fewer load round trips and
// barriers per tile (K up to 1024 in late DenseNet blocks).  The data
// gradient (K = 128, N up to 1024, epilogue-bound) keeps 32: wider chunks
// made it slower.
constexpr int kRowsBKDirect = 64;
template <int SP> constexpr int rows_bk() { return SP == SP_FWD_BNRELU ? kRowsBKDirect : kRowsBK; }

template <typename T, int TAPS, int BM, int BN, int WM, int WN, int SP>
__global__ __launch_bounds__(kThreads) void k_conv_rows(RowsParams p)
{
    static_assert(SP == SP_RUNTIME || (TAPS == 1 && sizeof(T) == 2), "specialised cases are bf16 1x1");
    constexpr int BK = rows_bk<SP>();
    using Cfg = RowsCfg<T, TAPS, BM, BN, BK>;
    using M = Mfma<T>;
    constexpr int TM = BM / (WM * 16), TN = BN / (WN * 16);
    constexpr int VEC = Cfg::VEC, ASTR = Cfg::ASTR, VPR = BK / VEC;
    static_assert(WM * WN == 4, "four waves");
    static_assert(TM * WM * 16 == BM && TN * WN * 16 == BN, "tile");

    extern __shared__ __align__(16) unsigned char smem[];
    T *As = reinterpret_cast<T *>(smem);
    T *Bs = As + Cfg::A_ELEMS;
    float *coef = reinterpret_cast<float *>(smem + Cfg::LDS);

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WN, wn = wave % WN;
    const int mt = xcd_remap(blockIdx.x, gridDim.x);
    const int nt = blockIdx.y;
    const int64_t m = p.m;
    const int64_t p0 = (int64_t)mt * BM;
    const int n0 = nt * BN;
    const int H = p.h, W = p.w, K = p.K, N = p.N;
    const int halo = TAPS == 9 ? W + 1 : 0;
    const int arows = BM + 2 * halo;

    // per-channel prologue coefficients for all K channels; float32 data also
    // keeps the centre K (bn_centre) in coef[3 K + c]: x stands for x - K below
    constexpr bool kF32 = sizeof(T) == 4;
    auto kcen = [&](int c) __attribute__((always_inline)) {
        if constexpr (kF32) return coef[3 * K + c];
        else return 0.f;
    };
    // (CU channels per thread per pass, their loads at clamped indices issued
    // together before any use: one memory round trip per pass)
    constexpr int CU = 4;
    if (p.pro == PRO_BNRELU || p.pro == PRO_BNRELU_POOL || p.pro == PRO_BNADDRELU) {
        for (int cb = tid; cb < K; cb += CU * kThreads) {   // y = x c0 + c1
            float g[CU], b[CU], mu[CU], rs[CU], kc[CU];
            #pragma unroll
            for (int u = 0; u < CU; u++) {
                const int c = min(cb + u * kThreads, K - 1);
                g[u] = p.p_gamma[c]; b[u] = p.p_beta[c]; mu[u] = p.p_mean[c]; rs[u] = p.p_rstd[c];
                kc[u] = bn_centre<T>(p.p_ctr, c);
            }
            #pragma unroll
            for (int u = 0; u < CU; u++) {
                const int c = cb + u * kThreads;
                if (c < K) {
                    bn_coef(g[u], b[u], mu[u], rs[u], coef[K + c], coef[2 * K + c]);
                    if constexpr (kF32) coef[3 * K + c] = kc[u];
                }
            }
        }
    } else if (p.pro == PRO_BNGRAD) {
        const float inv_m = 1.0f / (float)m;
        const bool split = p.p_split != 0;
        for (int cb = tid; cb < K; cb += CU * kThreads) {
            float g[CU], mu[CU], rs[CU], dg[CU], db[CU], kc[CU];
            #pragma unroll
            for (int u = 0; u < CU; u++) {
                const int c = min(cb + u * kThreads, K - 1);
                mu[u] = p.p_mean[c]; rs[u] = p.p_rstd[c];
                g[u] = split ? p.p_alpha[c] : p.p_gamma[c];
                dg[u] = split ? p.p_betap[c] : p.p_dgamma[c];
                db[u] = split ? 0.f : p.p_dbeta[c];
                kc[u] = bn_centre<T>(p.p_ctr, c);
            }
            #pragma unroll
            for (int u = 0; u < CU; u++) {
                const int c = cb + u * kThreads;
                if (c < K) {
                    deferred_coef_of(p.p_split, inv_m, g[u], mu[u], rs[u], dg[u], db[u], coef[c], coef[K + c],
                                     coef[2 * K + c]);
                    if constexpr (kF32) coef[3 * K + c] = kc[u];
                }
            }
        }
    }

    // geometry of this lane's output rows
    int hh[TM], ww[TM];
    bool rv[TM];
    for (int rb = 0; rb < TM; rb++) {
        const int64_t pp = p0 + wm * TM * 16 + rb * 16 + (lane & 15);
        rv[rb] = pp < m;
        ww[rb] = (int)(pp % W);
        hh[rb] = (int)((pp / W) % H);
    }

    f32x4 acc[TM][TN];
    for (int rb = 0; rb < TM; rb++)
        for (int cb = 0; cb < TN; cb++) acc[rb][cb] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int nchunks = (K + BK - 1) / BK;
    const T *asrc = reinterpret_cast<const T *>(p.a);
    const T *asrc2 = reinterpret_cast<const T *>(p.a2);
    __syncthreads();

    if constexpr (TAPS == 1) {
        if (SP != SP_RUNTIME || p.buf32) {
            // 1x1 with every operand span below 2^31 bytes: the next chunk's A
            // rows and weights are loaded into registers (raw buffer loads,
            // out-of-range offsets read zeros) while the matrix cores work on
            // the current chunk.  A slot j of this thread is row i / VPR,
            // channel vector i % VPR of the chunk (i = tid + j kThreads); its
            // source pixel is fixed for the whole tile.
            constexpr int NA = (BM * VPR + kThreads - 1) / kThreads, NB = (BN * VPR + kThreads - 1) / kThreads;
            const int pro = SP == SP_FWD_BNRELU ? PRO_BNRELU : (SP == SP_DGRAD_BNGRAD ? PRO_BNGRAD : p.pro);
            const bool pool = pro == PRO_POOLUP;
            const int64_t src_rows = pool ? m / 4 : m;
            const __amdgpu_buffer_rsrc_t abuf = buf_view(p.a, (uint32_t)(((src_rows - 1) * p.a_ldc + K) * sizeof(T)));
            const __amdgpu_buffer_rsrc_t a2buf =
                buf_view(pro == PRO_BNGRAD ? p.a2 : p.a,
                         pro == PRO_BNGRAD ? (uint32_t)(((m - 1) * p.a2_ldc + K) * sizeof(T)) : 0u);
            // weights: packed [nt][chunk][n][32 k], or (bf16, wdirect) the caller's
            // [k][n] (forward: staged as rows of k, fragments by transposing
            // reads) or [n][k] (data gradient: rows of n, as the packed layout)
            constexpr bool kTr = std::is_same<T, bf16_t>::value;
            const bool direct = SP != SP_RUNTIME || (kTr && p.wdirect);
            const bool dfwd = SP == SP_FWD_BNRELU || (SP == SP_RUNTIME && direct && !p.wtrans);
            constexpr int BP = BN + 8;                                // pitch of the [k][n] staging
            const __amdgpu_buffer_rsrc_t wbuf =
                direct ? buf_view(p.wraw, (uint32_t)((int64_t)K * N * sizeof(T)))
                       : buf_view(p.wpack, (uint32_t)((int64_t)gridDim.y * nchunks * BN * BK * sizeof(T)));
            const int a_ldc = (int)p.a_ldc, a2_ldc = (int)p.a2_ldc;
            int apix[NA], arow[NA], avec[NA];
            #pragma unroll
            for (int j = 0; j < NA; j++) {
                const int i = tid + j * kThreads;
                arow[j] = i / VPR;
                avec[j] = i % VPR;
                const int64_t pp = p0 + arow[j];
                int64_t q = pp;
                if (pool) {
                    const int64_t img = pp / ((int64_t)H * W);
                    const int rem = (int)(pp - img * H * W);
                    const int y = rem / W, x = rem - y * W;
                    q = (img * (H / 2) + y / 2) * (W / 2) + x / 2;
                }
                apix[j] = pp < m && i < BM * VPR ? (int)q : -1;
            }
            vec16 ra[NA], rx[NA], rw[NB];
            auto load_chunk = [&](int ch) __attribute__((always_inline)) {
                const int c0 = ch * BK;
                #pragma unroll
                for (int j = 0; j < NA; j++) {
                    const int c = c0 + avec[j] * VEC;
                    const bool ok = apix[j] >= 0 && c < K;
                    ra[j] = bld16(abuf, ok ? (uint32_t)(apix[j] * a_ldc + c) * (uint32_t)sizeof(T) : kBufOff);
                    if (pro == PRO_BNGRAD)
                        rx[j] = bld16(a2buf, ok ? (uint32_t)(apix[j] * a2_ldc + c) * (uint32_t)sizeof(T) : kBufOff);
                }
                const uint32_t wofs = (uint32_t)(((int64_t)nt * nchunks + ch) * (BN * BK));
                #pragma unroll
                for (int j = 0; j < NB; j++) {
                    const int i = tid + j * kThreads;
                    uint32_t off = kBufOff;
                    if (dfwd) {                       // row k = i / (BN / VEC) of [k][n]
                        const int k = c0 + i / (BN / VEC), nn = n0 + (i % (BN / VEC)) * VEC;
                        if (i < BN * VPR && k < K && nn < N) off = (uint32_t)(k * N + nn) * (uint32_t)sizeof(T);
                    } else if (direct) {              // row n = i / VPR of [n][k]
                        const int nn = n0 + i / VPR, k = c0 + (i % VPR) * VEC;
                        if (i < BN * VPR && nn < N && k < K) off = (uint32_t)(nn * K + k) * (uint32_t)sizeof(T);
                    } else if (i < BN * VPR) {
                        off = (wofs + (uint32_t)((i / VPR) * BK + (i % VPR) * VEC)) * (uint32_t)sizeof(T);
                    }
                    rw[j] = bld16(wbuf, off);
                }
            };
            // every slot of a thread holds the same channel vector of a chunk
            // (kThreads is a multiple of VPR): its coefficients are read once
            // per chunk, not once per slot
            static_assert(kThreads % VPR == 0, "slot channels");
            auto store_chunk = [&](int ch) __attribute__((always_inline)) {
                const int c0 = ch * BK;
                const int cv = c0 + (tid % VPR) * VEC, cc = cv < K ? cv : 0;
                float k0[VEC], k1[VEC], k2[VEC], kc[VEC];
                if (pro == PRO_BNRELU || pro == PRO_BNGRAD) {
                    #pragma unroll
                    for (int e = 0; e < VEC; e++) {
                        k0[e] = coef[cc + e];
                        k1[e] = coef[K + cc + e];
                        k2[e] = coef[2 * K + cc + e];
                        kc[e] = kcen(cc + e);
                    }
                }
                #pragma unroll
                for (int j = 0; j < NA; j++) {
                    const int c = c0 + avec[j] * VEC;
                    vec16 out = ra[j];
                    if (pro == PRO_BNRELU) {
                        float f[VEC];
                        Elem<T>::unpack(ra[j], f);
                        #pragma unroll
                        for (int e = 0; e < VEC; e++) {
                            const float t = bn_lin(f[e] - kc[e], k1[e], k2[e]);
                            f[e] = t > 0.f ? t : 0.f;
                        }
                        out = Elem<T>::pack(f);
                    } else if (pro == PRO_BNGRAD) {
                        float d[VEC], x[VEC];
                        Elem<T>::unpack(ra[j], d);
                        Elem<T>::unpack(rx[j], x);
                        #pragma unroll
                        for (int e = 0; e < VEC; e++)
                            d[e] = __builtin_fmaf(k0[e], d[e], __builtin_fmaf(k1[e], x[e] - kc[e], k2[e]));
                        out = Elem<T>::pack(d);
                    } else if (pro == PRO_RELU) {
                        float f[VEC];
                        Elem<T>::unpack(ra[j], f);
                        #pragma unroll
                        for (int e = 0; e < VEC; e++) f[e] = f[e] > 0.f ? f[e] : 0.f;
                        out = Elem<T>::pack(f);
                    } else if (pool) {
                        float f[VEC];
                        Elem<T>::unpack(ra[j], f);
                        #pragma unroll
                        for (int e = 0; e < VEC; e++) f[e] *= 0.25f;
                        out = Elem<T>::pack(f);
                    }
                    // rows past the tensor and channels past K are zero (not bn(0))
                    const bool valid = apix[j] >= 0 && c < K;
                    #pragma unroll
                    for (int w4 = 0; w4 < 4; w4++) out.u[w4] = valid ? out.u[w4] : 0u;
                    if (tid + j * kThreads < BM * VPR)
                        *reinterpret_cast<vec16 *>(As + arow[j] * ASTR + avec[j] * VEC) = out;
                }
                #pragma unroll
                for (int j = 0; j < NB; j++) {
                    const int i = tid + j * kThreads;
                    if (i < BN * VPR) {
                        T *dst = dfwd ? Bs + (i / (BN / VEC)) * BP + (i % (BN / VEC)) * VEC
                                      : Bs + (i / VPR) * ASTR + (i % VPR) * VEC;
                        *reinterpret_cast<vec16 *>(dst) = rw[j];
                    }
                }
            };
            load_chunk(0);
            for (int ch = 0; ch < nchunks; ch++) {
                store_chunk(ch);
                __syncthreads();
                if (ch + 1 < nchunks) load_chunk(ch + 1);
                for (int ks = 0; ks < BK / M::KSTEP; ks++) {
                    const int kofs = ks * M::KSTEP + (lane >> 4) * M::KPL;
                    typename M::frag b[TN];
                    if constexpr (kTr) {
                        if (dfwd) {                   // 8 consecutive k of one column of [k][n]
                            const bf16_t *bb = reinterpret_cast<const bf16_t *>(Bs) +
                                               (ks * M::KSTEP + 8 * (lane >> 4) + ((lane & 15) >> 2)) * BP +
                                               4 * (lane & 3) + wn * TN * 16;
                            #pragma unroll
                            for (int cb = 0; cb < TN; cb++) b[cb] = tr_frag(bb + cb * 16, BP);
                        } else {
                            #pragma unroll
                            for (int cb = 0; cb < TN; cb++)
                                b[cb] = M::load(Bs + (wn * TN * 16 + cb * 16 + (lane & 15)) * ASTR + kofs);
                        }
                    } else {
                        #pragma unroll
                        for (int cb = 0; cb < TN; cb++)
                            b[cb] = M::load(Bs + (wn * TN * 16 + cb * 16 + (lane & 15)) * ASTR + kofs);
                    }
                    #pragma unroll
                    for (int rb = 0; rb < TM; rb++) {
                        const typename M::frag a = M::load(As + (wm * TM * 16 + rb * 16 + (lane & 15)) * ASTR + kofs);
                        #pragma unroll
                        for (int cb = 0; cb < TN; cb++) M::mma(acc[rb][cb], a, b[cb]);
                    }
                }
                __syncthreads();
            }
        }
    }
    for (int ch = 0; ch < ((TAPS == 1 && (SP != SP_RUNTIME || p.buf32)) ? 0 : nchunks); ch++) {
        const int c0 = ch * BK;
        // ---- stage A (prologue applied, zero outside the tensor) ----
        for (int i = tid; i < arows * VPR; i += kThreads) {
            const int r = i / VPR, v = i % VPR;
            const int64_t pp = p0 - halo + r;
            const int c = c0 + v * VEC;
            vec16 out = zero16();
            if (pp >= 0 && pp < m && c < K) {
                if (p.pro == PRO_NONE) {
                    out = ldg16(asrc + pp * p.a_ldc + c);
                } else if (p.pro == PRO_BNRELU) {
                    float f[VEC];
                    Elem<T>::unpack(ldg16(asrc + pp * p.a_ldc + c), f);
                    for (int e = 0; e < VEC; e++) {
                        const float t = bn_lin(f[e] - kcen(c + e), coef[K + c + e], coef[2 * K + c + e]);
                        f[e] = t > 0.f ? t : 0.f;
                    }
                    out = Elem<T>::pack(f);
                    if (p.side && nt == 0 && r >= halo && r < halo + BM)
                        stg16(reinterpret_cast<T *>(p.side) + pp * p.side_ldc + c, out);
                } else if (p.pro == PRO_BNGRAD) {
                    float d[VEC], x[VEC];
                    Elem<T>::unpack(ldg16(asrc + pp * p.a_ldc + c), d);
                    Elem<T>::unpack(ldg16(asrc2 + pp * p.a2_ldc + c), x);
                    for (int e = 0; e < VEC; e++)
                        d[e] = __builtin_fmaf(coef[c + e], d[e],
                                              __builtin_fmaf(coef[K + c + e], x[e] - kcen(c + e), coef[2 * K + c + e]));
                    out = Elem<T>::pack(d);
                } else if (p.pro == PRO_RELU) {
                    float f[VEC];
                    Elem<T>::unpack(ldg16(asrc + pp * p.a_ldc + c), f);
                    for (int e = 0; e < VEC; e++) f[e] = f[e] > 0.f ? f[e] : 0.f;
                    out = Elem<T>::pack(f);
                } else if (p.pro == PRO_BNADDRELU) {
                    float f[VEC], id[VEC];
                    Elem<T>::unpack(ldg16(asrc + pp * p.a_ldc + c), f);
                    Elem<T>::unpack(ldg16(asrc2 + pp * p.a2_ldc + c), id);
                    for (int e = 0; e < VEC; e++)
                        f[e] = __builtin_fmaxf(bn_lin(f[e] - kcen(c + e), coef[K + c + e], coef[2 * K + c + e]) + id[e], 0.f);
                    out = Elem<T>::pack(f);
                    if (nt == 0) stg16(reinterpret_cast<T *>(p.side) + pp * p.side_ldc + c, out);
                } else if (p.pro == PRO_BNRELU_POOL) {
                    const int ho = H / 2, wo = W / 2;
                    const int64_t img = pp / ((int64_t)ho * wo);
                    const int rem = (int)(pp - img * ho * wo);
                    const int y = rem / wo, x = rem - y * wo;
                    const int64_t p00 = (img * H + 2 * y) * W + 2 * x;
                    float acc[VEC];
                    for (int e = 0; e < VEC; e++) acc[e] = 0.f;
                    for (int f4 = 0; f4 < 4; f4++) {
                        float f[VEC];
                        Elem<T>::unpack(ldg16(asrc + (p00 + (f4 >> 1) * W + (f4 & 1)) * p.a_ldc + c), f);
                        for (int e = 0; e < VEC; e++)
                            acc[e] += __builtin_fmaxf(bn_lin(f[e] - kcen(c + e), coef[K + c + e], coef[2 * K + c + e]), 0.f);
                    }
                    for (int e = 0; e < VEC; e++) acc[e] *= 0.25f;
                    out = Elem<T>::pack(acc);
                } else {  // PRO_POOLUP
                    const int64_t img = pp / ((int64_t)H * W);
                    const int rem = (int)(pp - img * H * W);
                    const int y = rem / W, x = rem - y * W;
                    const int64_t q = (img * (H / 2) + y / 2) * (W / 2) + x / 2;
                    float f[VEC];
                    Elem<T>::unpack(ldg16(asrc + q * p.a_ldc + c), f);
                    for (int e = 0; e < VEC; e++) f[e] *= 0.25f;
                    out = Elem<T>::pack(f);
                }
            }
            *reinterpret_cast<vec16 *>(As + r * ASTR + v * VEC) = out;
        }
        // ---- stage B: all taps of this chunk (packed, zero-padded) ----
        const T *wsrc = reinterpret_cast<const T *>(p.wpack) + ((int64_t)nt * nchunks + ch) * (TAPS * BN * BK);
        for (int i = tid; i < TAPS * BN * VPR; i += kThreads) {
            const int row = i / VPR, v = i % VPR;
            *reinterpret_cast<vec16 *>(Bs + row * ASTR + v * VEC) = ldg16(wsrc + row * BK + v * VEC);
        }
        __syncthreads();
        // ---- matrix cores ----
        for (int tap = 0; tap < TAPS; tap++) {
            const int dh = TAPS == 9 ? tap / 3 - 1 : 0, dw = TAPS == 9 ? tap % 3 - 1 : 0;
            const int off = dh * W + dw;
            for (int ks = 0; ks < BK / M::KSTEP; ks++) {
                const int kofs = ks * M::KSTEP + (lane >> 4) * M::KPL;
                typename M::frag b[TN];
                for (int cb = 0; cb < TN; cb++)
                    b[cb] = M::load(Bs + (tap * BN + wn * TN * 16 + cb * 16 + (lane & 15)) * ASTR + kofs);
                for (int rb = 0; rb < TM; rb++) {
                    const bool ok = rv[rb] && (unsigned)(hh[rb] + dh) < (unsigned)H &&
                                    (unsigned)(ww[rb] + dw) < (unsigned)W;
                    const int lrow = wm * TM * 16 + rb * 16 + (lane & 15) + halo + off;
                    typename M::frag a = M::load(As + lrow * ASTR + kofs);
                    if (!ok) a = M::zero();
                    for (int cb = 0; cb < TN; cb++) M::mma(acc[rb][cb], a, b[cb]);
                }
            }
        }
        __syncthreads();
    }

    // ---- epilogue: accumulators -> LDS tile (storage type) ----
    T *Cs = reinterpret_cast<T *>(smem);
    for (int rb = 0; rb < TM; rb++)
        for (int cb = 0; cb < TN; cb++)
            for (int i = 0; i < 4; i++) {
                const int row = wm * TM * 16 + rb * 16 + (lane >> 4) * 4 + i;
                const int col = wn * TN * 16 + cb * 16 + (lane & 15);
                Cs[row * Cfg::CSTR + col] = to_store<T>(acc[rb][cb][i]);
            }
    __syncthreads();

    constexpr int VPRO = BN / VEC, RSTEP = Cfg::RSTEP;
    const int v = tid % VPRO, r0 = tid / VPRO;
    const int n = n0 + v * VEC;
    const bool col_ok = n < N;
    float s1[VEC], s2[VEC], emu[VEC], ers[VEC], eg[VEC], eb[VEC], ek[VEC], es[VEC];
    for (int e = 0; e < VEC; e++) { s1[e] = 0.f; s2[e] = 0.f; ek[e] = 0.f; }
    const bool zsrc = p.epi == EPI_BNBWD && p.e_zsrc;
    bool zs = zsrc && col_ok;                     // this thread's vector reads z (else x)
    if (p.epi == EPI_BNBWD && col_ok) {
        // every parameter load first (a load inside a per-channel branch
        // becomes one memory round trip per channel)
        float ga[VEC], be[VEC];
        for (int e = 0; e < VEC; e++) {
            emu[e] = p.e_mean[n + e]; ers[e] = p.e_rstd[n + e]; ga[e] = p.e_gamma[n + e]; be[e] = p.e_beta[n + e];
            ek[e] = bn_centre<T>(p.e_ctr, n + e);
        }
        for (int e = 0; e < VEC; e++) zs = zs && ga[e] != 0.f;
        for (int e = 0; e < VEC; e++) {
            bn_coef(ga[e], be[e], emu[e], ers[e], eg[e], eb[e]);     // the forward's c0, c1
            es[e] = eg[e];                                          // summed-form scale
            if (zs) {                             // mask fma(z, 1, 0) > 0, xhat = (z - beta) / gamma
                emu[e] = be[e]; ers[e] = 1.0f / ga[e];
                eg[e] = 1.f; eb[e] = 0.f; ek[e] = 0.f;
            }
        }
    }
    const T *ex2s = reinterpret_cast<const T *>(p.ex2);
    if (p.epi == EPI_STATS)                       // statistics of y - shift
        for (int e = 0; e < VEC; e++) emu[e] = p.e_shift && col_ok ? p.e_shift[n + e] : 0.f;
    T *yout = reinterpret_cast<T *>(p.y);
    const T *exs = reinterpret_cast<const T *>(p.ex);
    if (col_ok) {
        for (int r = r0; r < BM; r += RSTEP) {
            const int64_t pp = p0 + r;
            if (pp >= m) break;
            const vec16 cv = *reinterpret_cast<const vec16 *>(Cs + r * Cfg::CSTR + v * VEC);
            T *dst = yout + pp * p.y_ldc + n;
            if (p.epi == EPI_STORE) {
                if (p.accumulate) {
                    float f[VEC], old[VEC];
                    Elem<T>::unpack(cv, f);
                    Elem<T>::unpack(ldg16(dst), old);
                    for (int e = 0; e < VEC; e++) f[e] += old[e];
                    stg16(dst, Elem<T>::pack(f));
                } else {
                    stg16(dst, cv);
                }
            } else if (p.epi == EPI_STATS) {
                float f[VEC];
                Elem<T>::unpack(cv, f);
                stg16(dst, cv);
                for (int e = 0; e < VEC; e++) { const float d = f[e] - emu[e]; s1[e] += d; s2[e] += d * d; }
            } else if (p.epi == EPI_RELUMASK) {
                float f[VEC], yv[VEC];
                Elem<T>::unpack(cv, f);
                Elem<T>::unpack(ldg16(exs + pp * p.ex_ldc + n), yv);
                for (int e = 0; e < VEC; e++) f[e] = yv[e] > 0.f ? f[e] : 0.f;
                stg16(dst, Elem<T>::pack(f));
            } else {
                float f[VEC], x[VEC], old[VEC];
                Elem<T>::unpack(cv, f);
                Elem<T>::unpack(ldg16(zsrc && !zs ? ex2s + pp * p.ex2_ldc + n : exs + pp * p.ex_ldc + n), x);
                if (p.e_scale && p.accumulate) Elem<T>::unpack(ldg16(dst), old);
                for (int e = 0; e < VEC; e++) {
                    const float xc = x[e] - ek[e];
                    const float xh = (xc - emu[e]) * ers[e];
                    const float d = bn_lin(xc, eg[e], eb[e]) > 0.f ? f[e] : 0.f;
                    s1[e] += d;
                    s2[e] += d * xh;
                    // summed-gradient form: gamma*rstd*dy, stored or added
                    f[e] = !p.e_scale ? d : (p.accumulate ? __builtin_fmaf(d, es[e], old[e]) : d * es[e]);
                }
                stg16(dst, Elem<T>::pack(f));
            }
        }
    }
    if (p.epi == EPI_STATS || p.epi == EPI_BNBWD) {
        __syncthreads();
        float *red = reinterpret_cast<float *>(smem);
        for (int e = 0; e < VEC; e++) {
            red[r0 * BN + v * VEC + e] = s1[e];
            red[(RSTEP + r0) * BN + v * VEC + e] = s2[e];
        }
        lds_colsum2(red, RSTEP, BN, BN, kThreads, tid, p.part + (int64_t)mt * 2 * N + n0,
                    p.part + (int64_t)mt * 2 * N + N + n0, N - n0);
    }
}

// ---------------------------------------------------------------------------
// Weight packing: W[kh][kw][ci][co] -> [ntile][chunk][tap][n][32] (GEMM order),
// zero outside the real K/N ranges.  transpose = 1 flips the taps and swaps
// ci/co (data-gradient operand).
template <typename T>
__global__ __launch_bounds__(kThreads) void k_pack_weights(const T *__restrict__ w, int taps, int c_in, int c_out,
                                                           int transpose, int bn, int nchunks, int64_t total,
                                                           T *__restrict__ out)
{
    for (int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * kThreads) {
        const int kk = (int)(idx % kRowsBK);
        int64_t t = idx / kRowsBK;
        const int nl = (int)(t % bn); t /= bn;
        const int tap = (int)(t % taps); t /= taps;
        const int ch = (int)(t % nchunks);
        const int ntile = (int)(t / nchunks);
        const int kc = ch * kRowsBK + kk, nn = ntile * bn + nl;
        T val = T(0);
        if (!transpose) {
            if (kc < c_in && nn < c_out) val = w[((int64_t)tap * c_in + kc) * c_out + nn];
        } else {
            if (kc < c_out && nn < c_in) val = w[((int64_t)(taps - 1 - tap) * c_in + nn) * c_out + kc];
        }
        out[idx] = val;
    }
}

// ------------------------------------------------------------- launchers ---
int64_t rows_mtiles(int dtype, int taps, int64_t m, int n_out)
{
    return ceil_div(m, rows_tile(dtype, taps, n_out, m).bm);
}

size_t rows_pack_bytes(int dtype, int taps, int K, int N)
{
    const RowsTile t = rows_tile(dtype, taps, N);
    const int64_t ntiles = ceil_div(N, t.bn), nchunks = ceil_div(K, kRowsBK);
    return (size_t)(ntiles * nchunks * taps * t.bn * kRowsBK) * (dtype == DT_BF16 ? 2 : 4);
}

hipError_t launch_pack_weights(int dtype, const void *w, int k, int c_in, int c_out, int transpose, void *wpack,
                               hipStream_t s)
{
    const int taps = k * k;
    const int K = transpose ? c_out : c_in, N = transpose ? c_in : c_out;
    const RowsTile t = rows_tile(dtype, taps, N);
    const int64_t ntiles = ceil_div(N, t.bn), nchunks = ceil_div(K, kRowsBK);
    const int64_t total = ntiles * nchunks * taps * t.bn * kRowsBK;
    const int grid = (int)(ceil_div(total, kThreads) < 1024 ? ceil_div(total, kThreads) : 1024);
    TraceScope tr(KC_SMALL, KID_PACK, s, (double)(taps * c_in * c_out + total) * (dtype == DT_BF16 ? 2 : 4), 0.0);
    if (dtype == DT_BF16)
        hipLaunchKernelGGL(k_pack_weights<bf16_t>, dim3(grid), dim3(kThreads), 0, s, (const bf16_t *)w, taps, c_in,
                           c_out, transpose, t.bn, (int)nchunks, total, (bf16_t *)wpack);
    else
        hipLaunchKernelGGL(k_pack_weights<float>, dim3(grid), dim3(kThreads), 0, s, (const float *)w, taps, c_in,
                           c_out, transpose, t.bn, (int)nchunks, total, (float *)wpack);
    return hipGetLastError();
}

// Algorithmic HBM bytes of one launch: each operand tensor read once, each
// output written once (weights once).
static double rows_algorithmic_bytes(const RowsParams &p)
{
    const double e = p.dtype == DT_BF16 ? 2.0 : 4.0, m = (double)p.m, K = p.K, N = p.N;
    double a = m * K;                                            // A operand
    if (p.pro == PRO_BNGRAD) a = 2.0 * m * K;                    // dy and x
    if (p.pro == PRO_POOLUP) a = m / 4.0 * K;                    // pooled gradient
    if (p.pro == PRO_BNRELU_POOL) a = 4.0 * m * K;               // four input pixels per window
    if (p.pro == PRO_BNADDRELU) a = 3.0 * m * K;                 // y and the identity read, the result written
    if (p.pro == PRO_BNRELU && p.side) a = 2.0 * m * K;          // x read, z written
    double out = m * N;                                          // output write
    if (p.epi == EPI_STORE && p.accumulate) out += m * N;        // read-modify-write
    if (p.epi == EPI_BNBWD || p.epi == EPI_RELUMASK) out += m * N;   // BN input / ReLU input read
    if (p.epi == EPI_BNBWD && p.e_scale && p.accumulate) out += m * N;  // summed gradient read
    return e * (a + out + (double)p.taps * K * N);
}

// every operand span of the tiled 1x1 kernel below 2^31 bytes (32-bit raw
// buffer offsets; the packed weights are at most ceil(N/32) * 32 * K_padded)
static bool rows_spans_fit(int dtype, int64_t m, int K, int N, int64_t a_ldc, int64_t a2_ldc, int pro)
{
    const int64_t lim = (int64_t)1 << 31, es = dtype == DT_BF16 ? 2 : 4;
    const int64_t src_rows = pro == PRO_POOLUP ? m / 4 : m;
    return (src_rows * a_ldc + K) * es < lim && (pro != PRO_BNGRAD || (m * a2_ldc + K) * es < lim) &&
           ceil_div(N, 32) * 32 * ceil_div(K, kRowsBK) * kRowsBK * es < lim;
}

bool rows_direct_weights(int dtype, int taps, int64_t m, int K, int N, int64_t a_ldc, int64_t a2_ldc, int pro,
                         bool side)
{
    return dtype == DT_BF16 && taps == 1 && pro != PRO_BNRELU_POOL && pro != PRO_BNADDRELU && !side &&
           rows_spans_fit(dtype, m, K, N, a_ldc, a2_ldc, pro);
}

template <typename T, int TAPS, int BM, int BN, int WM, int WN, int SP = SP_RUNTIME>
static hipError_t run_rows(const RowsParams &p, hipStream_t s)
{
    using Cfg = RowsCfg<T, TAPS, BM, BN, rows_bk<SP>()>;
    const int P = p.pro == PRO_BNRELU || p.pro == PRO_BNGRAD || p.pro == PRO_BNRELU_POOL || p.pro == PRO_BNADDRELU
                      ? (sizeof(T) == 4 ? 4 : 3) : 0;
    const size_t lds = Cfg::LDS + (size_t)P * p.K * sizeof(float);
    auto kern = k_conv_rows<T, TAPS, BM, BN, WM, WN, SP>;
    static bool attr_set = false;
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    dim3 grid((unsigned)ceil_div(p.m, BM), (unsigned)ceil_div(p.N, BN));
    TraceScope tr(KC_CONV, TAPS == 9 ? KID_CONV_3X3 : KID_CONV_1X1, s, rows_algorithmic_bytes(p),
                  2.0 * (double)p.m * TAPS * p.K * p.N);
    RowsParams q = p;
    q.buf32 = TAPS == 1 && p.pro != PRO_BNRELU_POOL && p.pro != PRO_BNADDRELU && !p.side &&
              rows_spans_fit(p.dtype, p.m, p.K, p.N, p.a_ldc, p.a2_ldc, p.pro);
    if (q.wdirect && (!q.buf32 || !p.wraw)) return hipErrorInvalidValue;   // unpacked weights need this path
    if (SP == SP_FWD_BNRELU && (!q.wdirect || p.wtrans || p.pro != PRO_BNRELU)) return hipErrorInvalidValue;
    if (SP == SP_DGRAD_BNGRAD && (!q.wdirect || !p.wtrans || p.pro != PRO_BNGRAD)) return hipErrorInvalidValue;
    hipLaunchKernelGGL(kern, grid, dim3(kThreads), lds, s, q);
    return hipGetLastError();
}

// Operands each prologue / epilogue mode reads must be present.
static bool rows_operands_ok(const RowsParams &p)
{
    if (!p.a || !(p.wdirect ? p.wraw : p.wpack) || !p.y) return false;
    if ((p.pro == PRO_BNRELU || p.pro == PRO_BNRELU_POOL || p.pro == PRO_BNADDRELU) && (!p.p_mean || !p.p_gamma || !p.p_rstd || !p.p_beta))
        return false;
    if (p.pro == PRO_BNADDRELU && (p.taps != 1 || !p.a2 || !p.side || p.wtrans || p.epi == EPI_BNBWD ||
                                   p.epi == EPI_RELUMASK))
        return false;
    if (p.pro == PRO_BNRELU_POOL && (p.taps != 1 || p.h % 2 || p.w % 2 || (int64_t)p.n * p.h * p.w != 4 * p.m ||
                                     p.wtrans || p.epi == EPI_BNBWD || p.epi == EPI_RELUMASK))
        return false;
    if (p.pro == PRO_BNGRAD && (!p.a2 || !p.p_mean || !p.p_rstd ||
                                (p.p_split ? (!p.p_alpha || !p.p_betap) : (!p.p_gamma || !p.p_dbeta || !p.p_dgamma))))
        return false;
    if ((p.epi == EPI_STATS || p.epi == EPI_BNBWD) && !p.part) return false;
    if (p.epi == EPI_BNBWD && (!p.ex || !p.e_mean || !p.e_rstd || !p.e_gamma || !p.e_beta)) return false;
    if (p.epi == EPI_RELUMASK && !p.ex) return false;
    if (p.side && p.pro != PRO_BNADDRELU &&
        (p.pro != PRO_BNRELU || p.wtrans || p.epi == EPI_BNBWD || p.epi == EPI_RELUMASK || p.wdirect))
        return false;
    if (p.e_zsrc && (p.epi != EPI_BNBWD || !p.ex2)) return false;
    if (p.taps == 9 && p.w > kRowsMaxW3) return false;
    return true;
}

hipError_t launch_conv_rows(const RowsParams &p, hipStream_t s)
{
    if (!rows_operands_ok(p)) return hipErrorInvalidValue;
    const RowsTile t = rows_tile(p.dtype, p.taps, p.N, p.m);
    if (p.dtype == DT_BF16) {
        if (p.taps == 1) {
            const bool dw = p.wdirect && rows_spans_fit(p.dtype, p.m, p.K, p.N, p.a_ldc, p.a2_ldc, p.pro);
            if (dw && p.pro == PRO_BNRELU && !p.wtrans) {
                if (t.bn == 32) return run_rows<bf16_t, 1, 128, 32, 4, 1, SP_FWD_BNRELU>(p, s);
                if (t.bn == 64) return run_rows<bf16_t, 1, 128, 64, 4, 1, SP_FWD_BNRELU>(p, s);
                if (t.bm == 32) return run_rows<bf16_t, 1, 32, 128, 2, 2, SP_FWD_BNRELU>(p, s);
                if (t.bm == 64) return run_rows<bf16_t, 1, 64, 128, 2, 2, SP_FWD_BNRELU>(p, s);
                return run_rows<bf16_t, 1, 128, 128, 2, 2, SP_FWD_BNRELU>(p, s);
            }
            if (dw && p.pro == PRO_BNGRAD && p.wtrans) {
                if (t.bn == 32) return run_rows<bf16_t, 1, 128, 32, 4, 1, SP_DGRAD_BNGRAD>(p, s);
                if (t.bn == 64) return run_rows<bf16_t, 1, 128, 64, 4, 1, SP_DGRAD_BNGRAD>(p, s);
                if (t.bm == 32) return run_rows<bf16_t, 1, 32, 128, 2, 2, SP_DGRAD_BNGRAD>(p, s);
                if (t.bm == 64) return run_rows<bf16_t, 1, 64, 128, 2, 2, SP_DGRAD_BNGRAD>(p, s);
                return run_rows<bf16_t, 1, 128, 128, 2, 2, SP_DGRAD_BNGRAD>(p, s);
            }
            if (t.bn == 32) return run_rows<bf16_t, 1, 128, 32, 4, 1>(p, s);
            if (t.bn == 64) return run_rows<bf16_t, 1, 128, 64, 4, 1>(p, s);
            if (t.bm == 32) return run_rows<bf16_t, 1, 32, 128, 2, 2>(p, s);
            if (t.bm == 64) return run_rows<bf16_t, 1, 64, 128, 2, 2>(p, s);
            return run_rows<bf16_t, 1, 128, 128, 2, 2>(p, s);
        }
        if (t.bn == 32) return run_rows<bf16_t, 9, 128, 32, 4, 1>(p, s);
        return run_rows<bf16_t, 9, 128, 64, 4, 1>(p, s);
    }
    if (p.taps == 1) {
        if (t.bn == 32) return run_rows<float, 1, 64, 32, 4, 1>(p, s);
        return run_rows<float, 1, 64, 64, 4, 1>(p, s);
    }
    if (t.bn == 32) return run_rows<float, 9, 64, 32, 4, 1>(p, s);
    return run_rows<float, 9, 64, 64, 4, 1>(p, s);
}

}  // namespace bnr
