// conv_wgrad.hip -- CONV weight gradient on the gfx950 matrix cores with the
// fission/fusion prologues on both operands.
//
//   dW[kh][kw][ci][co] = sum over pixels q of Z[q][ci] * G[q - off][co] * valid
//
// with off = (kh-1)*W + (kw-1) for 3x3 (0 for 1x1): the tap shift is applied
// to the gradient operand, so the Z operand is read unshifted.  valid is 1 when
// pixel q - off is the in-image neighbour of q for that tap (zero padding).
// Z is relu(bn(x)) recomputed from x (sub-BN2 recomputation, no stored
// activation), or x itself; G is a dense gradient, the deferred BN input
// gradient k*(dy - a - xhat*b) formed from (dy, x) on the fly, or the
// average-pooling gradient formed from the pooled gradient.
//
// GEMM view: M = 64 input channels (one 16-row block per wave) x taps of one
// filter row, N = output channels, K = pixels.  Pixels come in chunks of 64,
// staged transposed in LDS (channel-major, pixel-contiguous) so that a lane's
// 8 consecutive k values are one 16-byte read.  The pixel range is split S
// ways; each split writes a float32 partial tile and a fixed-order sum
// produces dW (deterministic).
#include "common.hpp"
#include "kernels.hpp"
#include "mfma.hpp"
#include "tiles.hpp"

namespace bnr {

template <typename T, int TPW, int COT>
struct WgCfg {
    static constexpr int VEC = Elem<T>::VEC;
    static constexpr int PAD = 16 / (int)sizeof(T);
    static constexpr int ZSTR = kWgBKP + PAD;
    static constexpr int HALO_MAX = TPW == 3 ? kRowsMaxW3 + 1 : 0;
    static constexpr int GCOLS = kWgBKP + 2 * HALO_MAX;
    static constexpr int GSTR = GCOLS + PAD;
    static constexpr size_t Z_BYTES = (size_t)kWgCIT * ZSTR * sizeof(T);
    static constexpr size_t G_BYTES = (size_t)COT * GSTR * sizeof(T);
};

template <typename T, int TPW, int COT>
__global__ __launch_bounds__(kThreads) void k_wgrad(WgradParams p, int ci_tiles, int kh_tiles, int co_tiles,
                                                   int64_t chunks_per_split, int64_t nchunks, int splits)
{
    using Cfg = WgCfg<T, TPW, COT>;
    using M = Mfma<T>;
    constexpr int VEC = Cfg::VEC, ZSTR = Cfg::ZSTR, GSTR = Cfg::GSTR;
    constexpr int TN = COT / 16;
    __shared__ __align__(16) T Zt[kWgCIT * ZSTR];
    __shared__ __align__(16) T Gt[COT * GSTR];
    __shared__ uint8_t flags[kWgBKP];
    __shared__ float zc[3][kWgCIT];
    __shared__ float gc[5][COT];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int n_out = ci_tiles * kh_tiles * co_tiles;
    const int lid = xcd_remap(blockIdx.x, gridDim.x);
    const int ot = lid % n_out, split = lid / n_out;
    const int co_t = ot % co_tiles, kh_t = (ot / co_tiles) % kh_tiles, ci_t = ot / (co_tiles * kh_tiles);
    const int ci0 = ci_t * kWgCIT, co0 = co_t * COT;
    const int H = p.h, W = p.w, C_in = p.c_in, C_out = p.c_out;
    const int64_t m = p.m;
    const int halo = TPW == 3 ? W + 1 : 0;
    const int dh = TPW == 3 ? kh_t - 1 : 0;

    // operand prologue coefficients for this tile's channels
    if (tid < kWgCIT) {
        const int c = ci0 + tid;
        if (p.a_mode == 1 && c < C_in) {
            zc[0][tid] = p.a_mean[c];
            zc[1][tid] = p.a_gamma[c] * p.a_rstd[c];
            zc[2][tid] = p.a_beta[c];
        }
    }
    if (tid < COT) {
        const int c = co0 + tid;
        if (p.gsrc == GB_BNGRAD && c < C_out) {
            const float inv_m = 1.0f / (float)m;
            gc[0][tid] = p.g_mean[c];
            gc[1][tid] = p.g_rstd[c];
            gc[2][tid] = p.g_gamma[c] * p.g_rstd[c];
            gc[3][tid] = p.g_dbeta[c] * inv_m;
            gc[4][tid] = p.g_dgamma[c] * inv_m;
        }
    }

    f32x4 acc[TPW][TN];
    for (int t = 0; t < TPW; t++)
        for (int cb = 0; cb < TN; cb++) acc[t][cb] = f32x4{0.f, 0.f, 0.f, 0.f};

    const T *xs = reinterpret_cast<const T *>(p.x);
    const T *gs = reinterpret_cast<const T *>(p.g);
    const T *gxs = reinterpret_cast<const T *>(p.gx);
    const int64_t ch_begin = (int64_t)split * chunks_per_split;
    const int64_t ch_end = min(nchunks, ch_begin + chunks_per_split);
    const int gcols = kWgBKP + 2 * halo;
    __syncthreads();

    for (int64_t ch = ch_begin; ch < ch_end; ch++) {
        const int64_t q0 = ch * kWgBKP;
        // ---- stage Z^T: 64 channels x 64 pixels, two pixels per item ----
        {
            constexpr int VPP = kWgCIT / VEC;                 // vectors per pixel
            constexpr int ITEMS = (kWgBKP / 2) * VPP;
            for (int i = tid; i < ITEMS; i += kThreads) {
                const int v = i % VPP, pr = i / VPP;
                const int cl = v * VEC, c = ci0 + cl;
                float f0[VEC], f1[VEC];
                for (int h2 = 0; h2 < 2; h2++) {
                    float *f = h2 ? f1 : f0;
                    const int64_t q = q0 + 2 * pr + h2;
                    if (q < m && c < C_in) {
                        Elem<T>::unpack(ldg16(xs + q * p.x_ldc + c), f);
                        if (p.a_mode == 1)
                            for (int e = 0; e < VEC; e++) {
                                const float t = (f[e] - zc[0][cl + e]) * zc[1][cl + e] + zc[2][cl + e];
                                f[e] = Elem<T>::round(t > 0.f ? t : 0.f);
                            }
                        else if (p.a_mode == 2)
                            for (int e = 0; e < VEC; e++) f[e] = f[e] > 0.f ? f[e] : 0.f;
                    } else {
                        for (int e = 0; e < VEC; e++) f[e] = 0.f;
                    }
                }
                for (int e = 0; e < VEC; e++) {
                    T *dst = Zt + (cl + e) * ZSTR + 2 * pr;
                    dst[0] = to_store<T>(f0[e]);
                    dst[1] = to_store<T>(f1[e]);
                }
            }
        }
        // ---- stage G^T with the tap halo: COT channels x gcols pixels ----
        {
            constexpr int VPP = COT / VEC;
            const int items = (gcols / 2) * VPP;
            for (int i = tid; i < items; i += kThreads) {
                const int v = i % VPP, pr = i / VPP;
                const int cl = v * VEC, c = co0 + cl;
                float f0[VEC], f1[VEC];
                for (int h2 = 0; h2 < 2; h2++) {
                    float *f = h2 ? f1 : f0;
                    const int64_t q = q0 - halo + 2 * pr + h2;
                    if (q >= 0 && q < m && c < C_out) {
                        if (p.gsrc == GB_DENSE) {
                            Elem<T>::unpack(ldg16(gs + q * p.g_ldc + c), f);
                        } else if (p.gsrc == GB_BNGRAD) {
                            float x[VEC];
                            Elem<T>::unpack(ldg16(gs + q * p.g_ldc + c), f);
                            Elem<T>::unpack(ldg16(gxs + q * p.gx_ldc + c), x);
                            for (int e = 0; e < VEC; e++) {
                                const float xh = (x[e] - gc[0][cl + e]) * gc[1][cl + e];
                                f[e] = Elem<T>::round(gc[2][cl + e] * (f[e] - gc[3][cl + e] - xh * gc[4][cl + e]));
                            }
                        } else {
                            const int64_t img = q / ((int64_t)H * W);
                            const int rem = (int)(q - img * H * W);
                            const int y = rem / W, xx = rem - y * W;
                            const int64_t qq = (img * (H / 2) + y / 2) * (W / 2) + xx / 2;
                            Elem<T>::unpack(ldg16(gs + qq * p.g_ldc + c), f);
                            for (int e = 0; e < VEC; e++) f[e] *= 0.25f;
                        }
                    } else {
                        for (int e = 0; e < VEC; e++) f[e] = 0.f;
                    }
                }
                for (int e = 0; e < VEC; e++) {
                    T *dst = Gt + (cl + e) * GSTR + 2 * pr;
                    dst[0] = to_store<T>(f0[e]);
                    dst[1] = to_store<T>(f1[e]);
                }
            }
        }
        // ---- border flags of the chunk's pixels (3x3 only) ----
        if (TPW == 3 && tid < kWgBKP) {
            const int64_t q = q0 + tid;
            uint8_t f = 0;
            if (q < m) {
                const int wq = (int)(q % W), hq = (int)((q / W) % H);
                f = 1 | (hq == 0 ? 2 : 0) | (hq == H - 1 ? 4 : 0) | (wq == 0 ? 8 : 0) | (wq == W - 1 ? 16 : 0);
            }
            flags[tid] = f;
        }
        __syncthreads();
        // ---- matrix cores ----
        for (int ks = 0; ks < kWgBKP / M::KSTEP; ks++) {
            const int kq = ks * M::KSTEP + (lane >> 4) * M::KPL;
            const typename M::frag a = M::load(Zt + (wave * 16 + (lane & 15)) * ZSTR + kq);
            for (int t = 0; t < TPW; t++) {
                if (TPW == 1) {
                    for (int cb = 0; cb < TN; cb++) {
                        const typename M::frag b = M::load(Gt + (cb * 16 + (lane & 15)) * GSTR + kq);
                        M::mma(acc[t][cb], a, b);
                    }
                } else {
                    const int dw = t - 1;
                    const int off = dh * W + dw;
                    const int bad = (dh == 1 ? 2 : (dh == -1 ? 4 : 0)) | (dw == 1 ? 8 : (dw == -1 ? 16 : 0));
                    bool ok[M::KPL];
                    for (int e = 0; e < M::KPL; e++) {
                        const int f = flags[kq + e];
                        ok[e] = (f & 1) && !(f & bad);
                    }
                    for (int cb = 0; cb < TN; cb++) {
                        const T *src = Gt + (cb * 16 + (lane & 15)) * GSTR + halo - off + kq;
                        typename M::frag b;
                        if constexpr (M::KPL == 8) {
                            uint32_t wv[4];
                            for (int e2 = 0; e2 < 4; e2++) {
                                const uint32_t lo = ok[2 * e2] ? (uint32_t)src[2 * e2] : 0u;
                                const uint32_t hi = ok[2 * e2 + 1] ? (uint32_t)src[2 * e2 + 1] : 0u;
                                wv[e2] = lo | (hi << 16);
                            }
                            b = M::from_words(wv);
                        } else {
                            b = ok[0] ? M::load(src) : M::zero();
                        }
                        M::mma(acc[t][cb], a, b);
                    }
                }
            }
        }
        __syncthreads();
    }

    // ---- partial tile (or dW directly when there is one split) ----
    float *dst = splits == 1 ? p.dw : p.part + (int64_t)split * p.k * p.k * C_in * C_out;
    for (int t = 0; t < TPW; t++) {
        const int tap = TPW == 3 ? kh_t * 3 + t : 0;
        for (int cb = 0; cb < TN; cb++)
            for (int i = 0; i < 4; i++) {
                const int ci = ci0 + wave * 16 + (lane >> 4) * 4 + i;
                const int co = co0 + cb * 16 + (lane & 15);
                if (ci < C_in && co < C_out) dst[((int64_t)tap * C_in + ci) * C_out + co] = acc[t][cb][i];
            }
    }
}

// ------------------------------------------------------------- launchers ---
size_t wgrad_ws_bytes(int dtype, int64_t m, int c_in, int c_out, int k)
{
    const WgradPlan pl = wgrad_plan(m, c_in, c_out, k, dtype == DT_BF16 ? 2 : 4);
    if (pl.splits <= 1) return 0;
    return (size_t)pl.splits * k * k * c_in * c_out * sizeof(float);
}

template <typename T, int TPW, int COT>
static hipError_t run_wgrad(const WgradParams &p, const WgradPlan &pl, hipStream_t s)
{
    const int64_t nchunks = ceil_div(p.m, kWgBKP);
    const int64_t blocks = (int64_t)pl.ci_tiles * pl.kh_tiles * pl.co_tiles * pl.splits;
    hipLaunchKernelGGL((k_wgrad<T, TPW, COT>), dim3((unsigned)blocks), dim3(kThreads), 0, s, p, pl.ci_tiles,
                       pl.kh_tiles, pl.co_tiles, pl.chunks_per_split, nchunks, (int)pl.splits);
    return hipGetLastError();
}

hipError_t launch_wgrad(const WgradParams &p, hipStream_t s)
{
    if (!p.x || !p.g || !p.dw) return hipErrorInvalidValue;
    if (p.a_mode == 1 && (!p.a_mean || !p.a_gamma || !p.a_rstd || !p.a_beta)) return hipErrorInvalidValue;
    if (p.gsrc == GB_BNGRAD && (!p.gx || !p.g_mean || !p.g_rstd || !p.g_gamma || !p.g_dbeta || !p.g_dgamma))
        return hipErrorInvalidValue;
    if (p.k == 3 && p.w > kRowsMaxW3) return hipErrorInvalidValue;
    const WgradPlan pl = wgrad_plan(p.m, p.c_in, p.c_out, p.k, p.dtype == DT_BF16 ? 2 : 4);
    if (pl.splits > 1 && !p.part) return hipErrorInvalidValue;
    hipError_t e;
    if (p.dtype == DT_BF16) {
        if (p.k == 1)
            e = pl.cot == 32 ? run_wgrad<bf16_t, 1, 32>(p, pl, s)
              : pl.cot == 64 ? run_wgrad<bf16_t, 1, 64>(p, pl, s) : run_wgrad<bf16_t, 1, 128>(p, pl, s);
        else
            e = pl.cot == 32 ? run_wgrad<bf16_t, 3, 32>(p, pl, s)
              : pl.cot == 64 ? run_wgrad<bf16_t, 3, 64>(p, pl, s) : run_wgrad<bf16_t, 3, 128>(p, pl, s);
    } else {
        if (p.k == 1)
            e = pl.cot == 32 ? run_wgrad<float, 1, 32>(p, pl, s)
              : pl.cot == 64 ? run_wgrad<float, 1, 64>(p, pl, s) : run_wgrad<float, 1, 128>(p, pl, s);
        else
            e = pl.cot == 32 ? run_wgrad<float, 3, 32>(p, pl, s)
              : pl.cot == 64 ? run_wgrad<float, 3, 64>(p, pl, s) : run_wgrad<float, 3, 128>(p, pl, s);
    }
    if (e != hipSuccess || pl.splits <= 1) return e;
    return launch_sum_partials(p.part, pl.splits, (int64_t)p.k * p.k * p.c_in * p.c_out, p.dw, s);
}

}  // namespace bnr
