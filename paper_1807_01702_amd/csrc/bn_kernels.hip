// bn_kernels.hip -- HBM-streaming BN kernels: per-channel reductions (the
// sub-BN1 statistics sweep and the backward sums), their float64 combine,
// the standalone BN input gradient, the unfused A/B kernels (normalise, ReLU,
// ReLU backward), 2x2 average pooling and a calibration copy.
//
// Layout of every sweep: a workgroup owns a block of pixel rows and up to 32
// 16-byte channel vectors of each row; thread (tx, ty) reads vector tx of rows
// ty, ty+RY, ... so each wave reads whole contiguous row segments (coalesced
// NHWC) and keeps its channels' per-thread sums in registers.
#include "common.hpp"
#include "kernels.hpp"
#include "tiles.hpp"
#include "trace.hpp"

namespace bnr {

// --------------------------------------------------------------------------
// Per-channel partial sums over a row block (MODE is a template argument so
// every load of a 4-row batch is issued before any arithmetic).
//   ST_SUMSQ : s1 = sum (x - K),      s2 = sum (x - K)^2  (mean/variance fusion; K = the
//              per-channel shift passed as `mean`, 0 if NULL)
//   ST_SUM   : s1 = sum x                                 (unfused mean sweep)
//   ST_SQDEV : s1 = sum (x - mean)^2                      (unfused variance sweep)
//   ST_DYX   : s1 = sum dy,           s2 = sum dy * xhat  (BN backward sums;
//              xhat = ((x - ctr) - mean) rstd, ctr the float32 centre, bn_centre)
// part[rb][0][c] = s1, part[rb][1][c] = s2 (float32).
template <typename T, int MODE>
__device__ __forceinline__ void stats_accum(const vec16 &v, const vec16 &d, const float *mu, const float *rs,
                                            const float *kc, float *s1, float *s2)
{
    constexpr int VEC = Elem<T>::VEC;
    float f[VEC];
    Elem<T>::unpack(v, f);
    if (MODE == ST_SUMSQ) {
        for (int i = 0; i < VEC; i++) { const float e = f[i] - mu[i]; s1[i] += e; s2[i] += e * e; }
    } else if (MODE == ST_SUM) {
        for (int i = 0; i < VEC; i++) s1[i] += f[i];
    } else if (MODE == ST_SQDEV) {
        for (int i = 0; i < VEC; i++) { const float e = f[i] - mu[i]; s1[i] += e * e; }
    } else {
        float g[VEC];
        Elem<T>::unpack(d, g);
        for (int i = 0; i < VEC; i++) { s1[i] += g[i]; s2[i] += g[i] * (((f[i] - kc[i]) - mu[i]) * rs[i]); }
    }
}

template <typename T, int MODE>
__global__ __launch_bounds__(kThreads) void k_stats_partial(
    const T *__restrict__ x, int64_t ldc, int64_t m, int C,
    const float *__restrict__ mean, const float *__restrict__ rstd,
    const T *__restrict__ dy, int64_t dy_ldc, int64_t rows_per_block, float *__restrict__ part,
    const float *__restrict__ ctr)
{
    constexpr int VEC = Elem<T>::VEC, U = 4;
    __shared__ float red[2][kThreads * VEC];
    const int cvec = C / VEC;
    const int vb = min(kStatsMaxVec, cvec - (int)blockIdx.y * kStatsMaxVec);
    const int ry = kThreads / vb;
    const int tid = threadIdx.x, tx = tid % vb, ty = tid / vb;
    const int c0 = ((int)blockIdx.y * kStatsMaxVec + tx) * VEC;
    float s1[VEC], s2[VEC], mu[VEC], rs[VEC], kc[VEC];
    for (int i = 0; i < VEC; i++) { s1[i] = 0.f; s2[i] = 0.f; mu[i] = 0.f; rs[i] = 1.f; kc[i] = 0.f; }
    if (ty < ry && MODE == ST_DYX)
        for (int i = 0; i < VEC; i++) kc[i] = bn_centre<T>(ctr, c0 + i);
    if (ty < ry && (MODE == ST_SQDEV || MODE == ST_DYX || (MODE == ST_SUMSQ && mean)))
        for (int i = 0; i < VEC; i++) mu[i] = mean[c0 + i];
    if (ty < ry && MODE == ST_DYX)
        for (int i = 0; i < VEC; i++) rs[i] = rstd[c0 + i];
    const int64_t r0 = (int64_t)blockIdx.x * rows_per_block;
    const int64_t r1 = min(m, r0 + rows_per_block);
    if (ty < ry) {
        int64_t r = r0 + ty;
        for (; r + (U - 1) * ry < r1; r += U * ry) {
            vec16 v[U], d[U];
            #pragma unroll
            for (int u = 0; u < U; u++) {
                v[u] = ldg16(x + (r + u * ry) * ldc + c0);
                d[u] = MODE == ST_DYX ? ldg16(dy + (r + u * ry) * dy_ldc + c0) : v[u];
            }
            #pragma unroll
            for (int u = 0; u < U; u++) stats_accum<T, MODE>(v[u], d[u], mu, rs, kc, s1, s2);
        }
        for (; r < r1; r += ry) {
            const vec16 v = ldg16(x + r * ldc + c0);
            const vec16 d = MODE == ST_DYX ? ldg16(dy + r * dy_ldc + c0) : v;
            stats_accum<T, MODE>(v, d, mu, rs, kc, s1, s2);
        }
    }
    const int nch = vb * VEC;
    if (ty < ry)
        for (int i = 0; i < VEC; i++) {
            red[0][ty * nch + tx * VEC + i] = s1[i];
            red[1][ty * nch + tx * VEC + i] = s2[i];
        }
    __syncthreads();
    if (tid < nch) {
        float a = 0.f, b = 0.f;
        for (int j = 0; j < ry; j++) { a += red[0][j * nch + tid]; b += red[1][j * nch + tid]; }
        const int c = (int)blockIdx.y * kStatsMaxVec * VEC + tid;
        float *p = part + (int64_t)blockIdx.x * 2 * C;
        p[c] = a;
        p[C + c] = b;
    }
}

// --------------------------------------------------------------------------
// Finalisation shared by the combine kernels: from the float64 sums a = s1,
// b = s2 of one channel write
//   FIN_MVF   : with K = st.shift (0 if NULL; the sums are of x - K):
//               mean = K + a/m, var = b/m - (a/m)^2 (clamped at 0), rstd
//   FIN_MEAN  : mean = a/m
//   (FIN_MVF, FIN_MEAN: st.mean_lo[c] = mean64 - (float)mean64, the low part)
//   FIN_VAR   : var = a/m, rstd            (two-pass variance)
//   (FIN_MVF, FIN_VAR: running statistics updated when st.rmean is set)
//   FIN_BWD   : dbeta = a, dgamma = b, and the summed-gradient terms of st
//               (SplitTerms) when st.alpha is set
__device__ __forceinline__ void stats_write(int mode, int c, double a, double b, int64_t m, float eps, float *mean,
                                            float *var, float *rstd, float *dbeta, float *dgamma,
                                            const SplitTerms &st)
{
    const double dm = (double)m;
    if (mode == FIN_MVF || mode == FIN_VAR) {
        double mu, v;
        if (mode == FIN_MVF) {                    // sums of x - K
            const double ms = a / dm;
            v = b / dm - ms * ms;
            if (v < 0.0) v = 0.0;
            mu = (st.shift ? (double)st.shift[c] : 0.0) + ms;
            const float mf = (float)mu;
            mean[c] = mf;
            if (st.mean_lo) st.mean_lo[c] = (float)(mu - (double)mf);
        } else {                                  // two-pass: a = sum (x - mean)^2
            v = a / dm;
            mu = st.rmean ? (double)mean[c] : 0.0;
        }
        if (var) var[c] = (float)v;
        rstd[c] = (float)(1.0 / sqrt(v + (double)eps));
        if (st.rmean) {
            const double mo = (double)st.momentum;
            st.rmean[c] = (float)((1.0 - mo) * (double)st.rmean[c] + mo * mu);
            if (st.rvar) st.rvar[c] = (float)((1.0 - mo) * (double)st.rvar[c] + mo * v * (dm > 1.0 ? dm / (dm - 1.0) : 1.0));
        }
    } else if (mode == FIN_MEAN) {
        const double mu = a / dm;
        const float mf = (float)mu;
        mean[c] = mf;
        if (st.mean_lo) st.mean_lo[c] = (float)(mu - (double)mf);
    } else {
        dbeta[c] = (float)a;
        dgamma[c] = (float)b;
        if (st.alpha) {
            float al0 = 0.f, bp0 = 0.f;           // (every load before any use: one round trip)
            const float g = st.gamma[c], r = st.rstd[c];
            if (st.accumulate) { al0 = st.alpha[c]; bp0 = st.betap[c]; }
            const double k = (double)g * (double)r;
            float al = (float)(-k * a / dm), bp = (float)(-k * b / dm);
            if (st.accumulate) { al += al0; bp += bp0; }
            st.alpha[c] = al;
            st.betap[c] = bp;
        }
    }
}

// One-kernel combine for up to kCombineOneMaxRows partial rows: workgroup =
// 8 channels x 32 row groups; thread (c, g) adds rows g, g+32, ... in float64
// (8 loads in flight), then the 32 group sums of a channel are added in a
// fixed order (deterministic).
__device__ __forceinline__ void combine_one_block(int bid, const float *__restrict__ part, int64_t R, int C,
                                                  int64_t m, int mode, float eps, float *mean, float *var,
                                                  float *rstd, float *dbeta, float *dgamma, const SplitTerms &st)
{
    __shared__ double red[2][32][8];
    const int tid = threadIdx.x, cl = tid & 7, g = tid >> 3;
    const int c = bid * 8 + cl;
    double a = 0.0, b = 0.0;
    if (c < C) {
        // rows past the last are read at the last row and selected away: no
        // branch around a load, so the 16 loads of a pass are in flight
        // together (a branch per load made one round trip each)
        const float *p = part + c;
        for (int64_t r = g; r < R; r += 8 * 32) {
            float va[8], vb[8];
            #pragma unroll
            for (int u = 0; u < 8; u++) {
                const int64_t rr = r + 32 * u, rc = rr < R ? rr : R - 1;
                va[u] = p[rc * 2 * C];
                vb[u] = p[rc * 2 * C + C];
            }
            #pragma unroll
            for (int u = 0; u < 8; u++) {
                const bool ok = r + 32 * u < R;
                va[u] = ok ? va[u] : 0.f;
                vb[u] = ok ? vb[u] : 0.f;
            }
            #pragma unroll
            for (int u = 0; u < 8; u++) { a += (double)va[u]; b += (double)vb[u]; }
        }
    }
    red[0][g][cl] = a;
    red[1][g][cl] = b;
    __syncthreads();
    if (g == 0 && c < C) {
        double sa = 0.0, sb = 0.0;
        for (int j = 0; j < 32; j++) { sa += red[0][j][cl]; sb += red[1][j][cl]; }
        stats_write(mode, c, sa, sb, m, eps, mean, var, rstd, dbeta, dgamma, st);
    }
}

__global__ __launch_bounds__(kThreads) void k_stats_combine_one(const float *__restrict__ part, int64_t R, int C,
                                                                int64_t m, int mode, float eps, float *mean,
                                                                float *var, float *rstd, float *dbeta, float *dgamma,
                                                                SplitTerms st)
{
    combine_one_block(blockIdx.x, part, R, C, m, mode, eps, mean, var, rstd, dbeta, dgamma, st);
}

// --------------------------------------------------------------------------
// Tail of a fused backward CONV call in one launch: the weight gradient's
// split-K sum and the BN-backward sums' combine (independent jobs).
//   workgroups [0, nb_sum): dw[i] = sum over the S partial tiles, one level:
//     a workgroup owns 16 consecutive float4 outputs; its 256 threads are 16
//     row groups x 16 outputs (row group q adds partials q, q+16, ... with
//     eight loads in flight), and the 16 row-group sums of an output are
//     added in a fixed order (deterministic);
//   workgroups [nb_sum, nb_sum + ceil(C/8)): the one-kernel statistics
//     combine (FIN_BWD, with the summed-gradient terms of st).
constexpr int kTailF4 = 16;
__global__ __launch_bounds__(kThreads) void k_bwd_tail(const float *__restrict__ wpart, int64_t S, int64_t len,
                                                       float *__restrict__ dw, int nb_sum,
                                                       const float *__restrict__ spart, int64_t R, int C, int64_t m,
                                                       float *dbeta, float *dgamma, SplitTerms st)
{
    if ((int)blockIdx.x >= nb_sum) {
        combine_one_block((int)blockIdx.x - nb_sum, spart, R, C, m, FIN_BWD, 0.f, nullptr, nullptr, nullptr, dbeta,
                          dgamma, st);
        return;
    }
    __shared__ float4 red[kThreads / kTailF4][kTailF4];
    const int tid = threadIdx.x, f = tid % kTailF4, q = tid / kTailF4;
    constexpr int QN = kThreads / kTailF4;
    const int64_t i4 = (int64_t)blockIdx.x * kTailF4 + f;
    const int64_t st4 = len / 4;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    if (i4 < st4) {
        // splits past the last are read at the last split and selected away:
        // no branch around a load, so the eight loads of a pass are in flight
        // together
        const float4 *p = reinterpret_cast<const float4 *>(wpart) + i4;
        for (int64_t r = q; r < S; r += 8 * QN) {
            float4 v[8];
            #pragma unroll
            for (int u = 0; u < 8; u++) {
                const int64_t rr = r + (int64_t)u * QN;
                v[u] = p[(rr < S ? rr : S - 1) * st4];
            }
            #pragma unroll
            for (int u = 0; u < 8; u++) {
                if (r + (int64_t)u * QN >= S) v[u] = make_float4(0.f, 0.f, 0.f, 0.f);
                acc.x += v[u].x; acc.y += v[u].y; acc.z += v[u].z; acc.w += v[u].w;
            }
        }
    }
    red[q][f] = acc;
    __syncthreads();
    if (q == 0 && i4 < st4) {
        float4 t = red[0][f];
        for (int j = 1; j < QN; j++) { const float4 a = red[j][f]; t.x += a.x; t.y += a.y; t.z += a.z; t.w += a.w; }
        reinterpret_cast<float4 *>(dw)[i4] = t;
    }
}

// --------------------------------------------------------------------------
// float64 combine of the partial tiles, in two kernels (the kernel boundary
// makes level 1 visible to level 2; no in-kernel fences).
// Level 1, grid (C/64, RS): workgroup (cg, rs) adds row blocks
// [rs*R/RS, (rs+1)*R/RS) of 64 channels (lane = channel, the 4 waves take
// interleaved rows, 8 loads in flight per lane) into float64 sums lvl1[rs].
__global__ __launch_bounds__(kThreads) void k_stats_combine1(const float *__restrict__ part, int64_t R, int C,
                                                             double *__restrict__ lvl1)
{
    __shared__ double red[2][4][64];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int c = blockIdx.x * 64 + lane;
    const int RS = gridDim.y, rs = blockIdx.y;
    const int64_t r0 = rs * R / RS, r1 = (rs + 1) * R / RS;
    double a = 0.0, b = 0.0;
    if (c < C) {
        // rows past the range are read at its last row and selected away (no
        // branch around a load)
        const float *p = part + c;
        for (int64_t r = r0 + wv; r < r1; r += 32) {
            float va[8], vb[8];
            #pragma unroll
            for (int u = 0; u < 8; u++) {
                const int64_t rr = r + 4 * u, rc = rr < r1 ? rr : r1 - 1;
                va[u] = p[rc * 2 * C];
                vb[u] = p[rc * 2 * C + C];
            }
            #pragma unroll
            for (int u = 0; u < 8; u++) {
                const bool ok = r + 4 * u < r1;
                va[u] = ok ? va[u] : 0.f;
                vb[u] = ok ? vb[u] : 0.f;
            }
            for (int u = 0; u < 8; u++) { a += (double)va[u]; b += (double)vb[u]; }
        }
    }
    red[0][wv][lane] = a;
    red[1][wv][lane] = b;
    __syncthreads();
    if (wv == 0 && c < C) {
        lvl1[((int64_t)rs * 2) * C + c] = red[0][0][lane] + red[0][1][lane] + red[0][2][lane] + red[0][3][lane];
        lvl1[((int64_t)rs * 2 + 1) * C + c] = red[1][0][lane] + red[1][1][lane] + red[1][2][lane] + red[1][3][lane];
    }
}

// Level 2: adds the RS level-1 sums of a channel in a fixed order
// (deterministic) and writes the statistics.
__global__ __launch_bounds__(kThreads) void k_stats_combine2(const double *__restrict__ lvl1, int RS, int C, int64_t m,
                                                             int mode, float eps, float *__restrict__ mean,
                                                             float *__restrict__ var, float *__restrict__ rstd,
                                                             float *__restrict__ dbeta, float *__restrict__ dgamma,
                                                             SplitTerms st)
{
    const int c = blockIdx.x * kThreads + threadIdx.x;
    if (c >= C) return;
    double a = 0.0, b = 0.0;
    for (int j = 0; j < RS; j++) {
        a += lvl1[((int64_t)j * 2) * C + c];
        b += lvl1[((int64_t)j * 2 + 1) * C + c];
    }
    stats_write(mode, c, a, b, m, eps, mean, var, rstd, dbeta, dgamma, st);
}

// --------------------------------------------------------------------------
// Element-wise passes over [m][C] views with per-channel parameters (MODE
// and ACC are template arguments so each row batch of four rows issues all
// its loads, including the accumulate read, before any arithmetic; the
// operands are streamed once, so the loads are non-temporal).
// (x - mean in every mode below stands for (x - ctr) - mean: ctr the float32
// centre, bn_centre, with mean given relative to it)
//   EW_DX      : out = gamma*rstd*(dy - dbeta/m - xhat*dgamma/m)  [+ out]
//   EW_APPLY   : out = gamma*(x-mean)*rstd + beta                  (unfused BN)
//   EW_RELU    : out = max(x, 0)                                   (unfused ReLU)
//   EW_RELUBWD : out = x2 > 0 ? x : 0   (x = dz, x2 = y)           (unfused ReLU bwd)
//   EW_BNADDRELU: out = max(gamma*(x-mean)*rstd + beta + x2, 0)    (residual BN + add + ReLU)
//   EW_ADDRELU : out = max(x + x2, 0)                              (unfused add + ReLU)
//   EW_SPLITDX : out = x + alpha + betap*(x2-mean)*rstd  [+ out]   (summed BN input
//                gradient; alpha is passed in dbeta's place, betap in dgamma's)
template <typename T, int MODE, bool ACC>
__global__ __launch_bounds__(kThreads) void k_elementwise(
    int64_t m, int C, const T *__restrict__ x, int64_t x_ldc, const T *__restrict__ x2,
    int64_t x2_ldc, const float *__restrict__ gamma, const float *__restrict__ beta,
    const float *__restrict__ mean, const float *__restrict__ rstd, const float *__restrict__ dgamma,
    const float *__restrict__ dbeta, T *__restrict__ out, int64_t out_ldc, int64_t rows_per_block,
    const float *__restrict__ ctr)
{
    constexpr int VEC = Elem<T>::VEC, U = 4;
    constexpr bool TWO = MODE == EW_DX || MODE == EW_RELUBWD || MODE == EW_BNADDRELU || MODE == EW_ADDRELU ||
                         MODE == EW_SPLITDX;
    const int cvec = C / VEC;
    const int vb = min(kStatsMaxVec, cvec - (int)blockIdx.y * kStatsMaxVec);
    const int ry = kThreads / vb;
    const int tid = threadIdx.x, tx = tid % vb, ty = tid / vb;
    if (ty >= ry) return;
    const int c0 = ((int)blockIdx.y * kStatsMaxVec + tx) * VEC;
    float p0[VEC], p1[VEC], p2[VEC], p3[VEC], p4[VEC], kc[VEC];
    const float inv_m = 1.0f / (float)m;
    for (int i = 0; i < VEC; i++) {
        const int c = c0 + i;
        p0[i] = p1[i] = p2[i] = p3[i] = p4[i] = 0.f;
        kc[i] = MODE == EW_DX || MODE == EW_APPLY || MODE == EW_BNADDRELU || MODE == EW_SPLITDX
                    ? bn_centre<T>(ctr, c) : 0.f;
        if (MODE == EW_DX) {
            p0[i] = gamma[c] * rstd[c];          // k
            p1[i] = dbeta[c] * inv_m;            // a
            p2[i] = dgamma[c] * inv_m;           // b
            p3[i] = mean[c];
            p4[i] = rstd[c];
        } else if (MODE == EW_APPLY) {
            p0[i] = gamma[c];
            p1[i] = beta[c];
            p2[i] = rstd[c];
            p3[i] = mean[c];
        } else if (MODE == EW_BNADDRELU) {
            bn_coef(gamma[c], beta[c], mean[c], rstd[c], p0[i], p1[i]);
        } else if (MODE == EW_SPLITDX) {
            p0[i] = dgamma[c] * rstd[c];         // betap * rstd
            p1[i] = dbeta[c] - p0[i] * mean[c];  // alpha - betap * rstd * mean
        }
    }
    auto row = [&](const vec16 &vx, const vec16 &v2, const vec16 &vo) __attribute__((always_inline)) {
        float f[VEC], g[VEC], o[VEC];
        Elem<T>::unpack(vx, f);
        if (TWO) Elem<T>::unpack(v2, g);
        if (MODE == EW_DX) {
            // f = dy, g = x
            for (int i = 0; i < VEC; i++) {
                const float xh = ((g[i] - kc[i]) - p3[i]) * p4[i];
                o[i] = p0[i] * (f[i] - p1[i] - xh * p2[i]);
            }
            if (ACC) {
                float old[VEC];
                Elem<T>::unpack(vo, old);
                for (int i = 0; i < VEC; i++) o[i] += old[i];
            }
        } else if (MODE == EW_APPLY) {
            for (int i = 0; i < VEC; i++) o[i] = p0[i] * (((f[i] - kc[i]) - p3[i]) * p2[i]) + p1[i];
        } else if (MODE == EW_RELU) {
            for (int i = 0; i < VEC; i++) o[i] = f[i] > 0.f ? f[i] : 0.f;
        } else if (MODE == EW_BNADDRELU) {
            for (int i = 0; i < VEC; i++) {
                const float t = bn_lin(f[i] - kc[i], p0[i], p1[i]) + g[i];
                o[i] = t > 0.f ? t : 0.f;
            }
        } else if (MODE == EW_ADDRELU) {
            for (int i = 0; i < VEC; i++) {
                const float t = f[i] + g[i];
                o[i] = t > 0.f ? t : 0.f;
            }
        } else if (MODE == EW_SPLITDX) {
            // f = summed gradient, g = x
            for (int i = 0; i < VEC; i++) o[i] = f[i] + __builtin_fmaf(p0[i], g[i] - kc[i], p1[i]);
            if (ACC) {
                float old[VEC];
                Elem<T>::unpack(vo, old);
                for (int i = 0; i < VEC; i++) o[i] += old[i];
            }
        } else {
            for (int i = 0; i < VEC; i++) o[i] = g[i] > 0.f ? f[i] : 0.f;
        }
        return Elem<T>::pack(o);
    };
    const int64_t r0 = (int64_t)blockIdx.x * rows_per_block;
    const int64_t r1 = min(m, r0 + rows_per_block);
    int64_t r = r0 + ty;
    for (; r + (U - 1) * ry < r1; r += U * ry) {
        vec16 vx[U], v2[U], vo[U];
        #pragma unroll
        for (int u = 0; u < U; u++) {
            const int64_t rr = r + u * ry;
            vx[u] = ldg16_stream(x + rr * x_ldc + c0);
            v2[u] = TWO ? ldg16_stream(x2 + rr * x2_ldc + c0) : vx[u];
            vo[u] = ACC ? ldg16_stream(out + rr * out_ldc + c0) : vx[u];
        }
        #pragma unroll
        for (int u = 0; u < U; u++) stg16(out + (r + u * ry) * out_ldc + c0, row(vx[u], v2[u], vo[u]));
    }
    for (; r < r1; r += ry) {
        const vec16 vx = ldg16_stream(x + r * x_ldc + c0);
        const vec16 v2 = TWO ? ldg16_stream(x2 + r * x2_ldc + c0) : vx;
        const vec16 vo = ACC ? ldg16_stream(out + r * out_ldc + c0) : vx;
        stg16(out + r * out_ldc + c0, row(vx, v2, vo));
    }
}

// --------------------------------------------------------------------------
// Backward of out = relu(bn(y) + identity) up to the BN reductions, in one
// sweep: gm = g * [out > 0] (the gradient of both the identity and the BN
// output), s1 = sum gm, s2 = sum gm * ((y - ctr) - mean) * rstd (ctr: the
// float32 centre, bn_centre).  Row blocks as in k_stats_partial.
template <typename T>
__global__ __launch_bounds__(kThreads) void k_addrelu_bwd(
    const T *g, int64_t g_ldc, const T *__restrict__ out, int64_t out_ldc, const T *__restrict__ y,
    int64_t y_ldc, int64_t m, int C, const float *__restrict__ mean, const float *__restrict__ rstd, T *gm,
    int64_t gm_ldc, int64_t rows_per_block, float *__restrict__ part, const float *__restrict__ ctr)
{
    constexpr int VEC = Elem<T>::VEC, U = 2;
    __shared__ float red[2][kThreads * VEC];
    const int cvec = C / VEC;
    const int vb = min(kStatsMaxVec, cvec - (int)blockIdx.y * kStatsMaxVec);
    const int ry = kThreads / vb;
    const int tid = threadIdx.x, tx = tid % vb, ty = tid / vb;
    const int c0 = ((int)blockIdx.y * kStatsMaxVec + tx) * VEC;
    float s1[VEC], s2[VEC], mu[VEC], rs[VEC], kc[VEC];
    for (int i = 0; i < VEC; i++) { s1[i] = 0.f; s2[i] = 0.f; mu[i] = 0.f; rs[i] = 0.f; kc[i] = 0.f; }
    if (ty < ry)
        for (int i = 0; i < VEC; i++) {
            mu[i] = mean[c0 + i]; rs[i] = rstd[c0 + i]; kc[i] = bn_centre<T>(ctr, c0 + i);
        }
    auto row = [&](const vec16 &vg, const vec16 &vo, const vec16 &vy, T *dst) __attribute__((always_inline)) {
        float fg[VEC], fo[VEC], fy[VEC];
        Elem<T>::unpack(vg, fg);
        Elem<T>::unpack(vo, fo);
        Elem<T>::unpack(vy, fy);
        for (int i = 0; i < VEC; i++) {
            const float d = fo[i] > 0.f ? fg[i] : 0.f;
            fg[i] = d;
            s1[i] += d;
            s2[i] += d * (((fy[i] - kc[i]) - mu[i]) * rs[i]);
        }
        stg16(dst, Elem<T>::pack(fg));
    };
    const int64_t r0 = (int64_t)blockIdx.x * rows_per_block;
    const int64_t r1 = min(m, r0 + rows_per_block);
    if (ty < ry) {
        int64_t r = r0 + ty;
        for (; r + (U - 1) * ry < r1; r += U * ry) {
            vec16 vg[U], vo[U], vy[U];
            #pragma unroll
            for (int u = 0; u < U; u++) {
                const int64_t rr = r + u * ry;
                vg[u] = ldg16(g + rr * g_ldc + c0);
                vo[u] = ldg16(out + rr * out_ldc + c0);
                vy[u] = ldg16(y + rr * y_ldc + c0);
            }
            #pragma unroll
            for (int u = 0; u < U; u++) row(vg[u], vo[u], vy[u], gm + (r + u * ry) * gm_ldc + c0);
        }
        for (; r < r1; r += ry)
            row(ldg16(g + r * g_ldc + c0), ldg16(out + r * out_ldc + c0), ldg16(y + r * y_ldc + c0),
                gm + r * gm_ldc + c0);
    }
    const int nch = vb * VEC;
    if (ty < ry)
        for (int i = 0; i < VEC; i++) {
            red[0][ty * nch + tx * VEC + i] = s1[i];
            red[1][ty * nch + tx * VEC + i] = s2[i];
        }
    __syncthreads();
    if (tid < nch) {
        float a = 0.f, b = 0.f;
        for (int j = 0; j < ry; j++) { a += red[0][j * nch + tid]; b += red[1][j * nch + tid]; }
        const int c = (int)blockIdx.y * kStatsMaxVec * VEC + tid;
        float *p = part + (int64_t)blockIdx.x * 2 * C;
        p[c] = a;
        p[C + c] = b;
    }
}

// --------------------------------------------------------------------------
// 2x2 / stride-2 average pooling: one thread per output 16-byte vector.
template <typename T>
__global__ __launch_bounds__(kThreads) void k_avgpool2(int n, int h, int w, int C, const T *__restrict__ x,
                                                       int64_t ldc, T *__restrict__ y, int64_t y_ldc)
{
    constexpr int VEC = Elem<T>::VEC;
    const int cvec = C / VEC, ho = h / 2, wo = w / 2;
    const int64_t total = (int64_t)n * ho * wo * cvec;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < total; i += (int64_t)gridDim.x * kThreads) {
        const int v = (int)(i % cvec);
        const int64_t op = i / cvec;
        const int ox = (int)(op % wo);
        const int64_t t = op / wo;
        const int oy = (int)(t % ho);
        const int64_t nn = t / ho;
        const int64_t ip = (nn * h + 2 * oy) * w + 2 * ox;
        float a[VEC], b[VEC], s[VEC];
        Elem<T>::unpack(ldg16(x + ip * ldc + v * VEC), s);
        Elem<T>::unpack(ldg16(x + (ip + 1) * ldc + v * VEC), a);
        for (int j = 0; j < VEC; j++) s[j] += a[j];
        Elem<T>::unpack(ldg16(x + (ip + w) * ldc + v * VEC), a);
        Elem<T>::unpack(ldg16(x + (ip + w + 1) * ldc + v * VEC), b);
        for (int j = 0; j < VEC; j++) s[j] = 0.25f * (s[j] + a[j] + b[j]);
        stg16(y + op * y_ldc + v * VEC, Elem<T>::pack(s));
    }
}

// Backward of the 2x2 pooling: every input pixel receives a quarter of its
// window's gradient.  One thread per input 16-byte vector.
template <typename T>
__global__ __launch_bounds__(kThreads) void k_avgpool2_bwd(int n, int h, int w, int C, const T *__restrict__ g,
                                                           int64_t g_ldc, T *__restrict__ gx, int64_t ldc)
{
    constexpr int VEC = Elem<T>::VEC;
    const int cvec = C / VEC;
    const int64_t total = (int64_t)n * h * w * cvec;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < total; i += (int64_t)gridDim.x * kThreads) {
        const int v = (int)(i % cvec);
        const int64_t ip = i / cvec;
        const int x = (int)(ip % w);
        const int64_t t = ip / w;
        const int y = (int)(t % h);
        const int64_t nn = t / h;
        const int64_t op = (nn * (h / 2) + y / 2) * (w / 2) + x / 2;
        float f[VEC];
        Elem<T>::unpack(ldg16(g + op * g_ldc + v * VEC), f);
        for (int j = 0; j < VEC; j++) f[j] *= 0.25f;
        stg16(gx + ip * ldc + v * VEC, Elem<T>::pack(f));
    }
}

// --------------------------------------------------------------------------
// Streaming copy (HBM calibration): each workgroup copies one contiguous
// range, four 16-byte vectors in flight per thread, non-temporal accesses.
__global__ __launch_bounds__(kThreads) void k_copy16(const vec16 *__restrict__ src, vec16 *__restrict__ dst,
                                                     int64_t nvec, int64_t per_block)
{
    const int64_t b0 = (int64_t)blockIdx.x * per_block;
    const int64_t b1 = b0 + per_block < nvec ? b0 + per_block : nvec;
    int64_t i = b0 + threadIdx.x;
    for (; i + 3 * kThreads < b1; i += 4 * kThreads) {
        vec16 t[4];
        #pragma unroll
        for (int u = 0; u < 4; u++)
            #pragma unroll
            for (int k = 0; k < 4; k++) t[u].u[k] = __builtin_nontemporal_load(&src[i + u * kThreads].u[k]);
        #pragma unroll
        for (int u = 0; u < 4; u++)
            #pragma unroll
            for (int k = 0; k < 4; k++) __builtin_nontemporal_store(t[u].u[k], &dst[i + u * kThreads].u[k]);
    }
    for (; i < b1; i += kThreads) dst[i] = src[i];
}

// Sum of S float32 partial tiles, in two kernels.  Level 1, grid
// (len/1024, SG): workgroup (i, g) adds splits [g*S/SG, (g+1)*S/SG) of 1024
// outputs (a float4 per thread, 4 loads in flight); level 2 adds the SG
// level-1 rows in a fixed order (deterministic).  With SG = 1 level 1 writes
// the result directly.
__global__ __launch_bounds__(kThreads) void k_sum_partials1(const float *__restrict__ part, int64_t S, int64_t len,
                                                            float *__restrict__ dst)
{
    const int SG = gridDim.y, g = blockIdx.y;
    const int64_t i4 = (int64_t)blockIdx.x * kThreads + threadIdx.x;     // float4 index
    if (i4 * 4 >= len) return;
    const int64_t s0 = g * S / SG, s1 = (g + 1) * S / SG;
    const float4 *p = reinterpret_cast<const float4 *>(part) + i4;
    const int64_t st = len / 4;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    int64_t s = s0;
    for (; s + 3 < s1; s += 4) {
        const float4 a = p[s * st], b = p[(s + 1) * st], c = p[(s + 2) * st], d = p[(s + 3) * st];
        acc.x += a.x; acc.y += a.y; acc.z += a.z; acc.w += a.w;
        acc.x += b.x; acc.y += b.y; acc.z += b.z; acc.w += b.w;
        acc.x += c.x; acc.y += c.y; acc.z += c.z; acc.w += c.w;
        acc.x += d.x; acc.y += d.y; acc.z += d.z; acc.w += d.w;
    }
    for (; s < s1; s++) {
        const float4 a = p[s * st];
        acc.x += a.x; acc.y += a.y; acc.z += a.z; acc.w += a.w;
    }
    reinterpret_cast<float4 *>(dst)[(int64_t)g * st + i4] = acc;
}

__global__ __launch_bounds__(kThreads) void k_sum_partials2(const float *__restrict__ lvl1, int SG, int64_t len,
                                                            float *__restrict__ out)
{
    const int64_t i4 = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (i4 * 4 >= len) return;
    const int64_t st = len / 4;
    float4 t = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int j = 0; j < SG; j++) {
        const float4 a = reinterpret_cast<const float4 *>(lvl1)[(int64_t)j * st + i4];
        t.x += a.x; t.y += a.y; t.z += a.z; t.w += a.w;
    }
    reinterpret_cast<float4 *>(out)[i4] = t;
}

// --------------------------------------------------------------- launchers --
static inline int grid_cap(int64_t want) { return (int)(want < 4096 ? (want < 1 ? 1 : want) : 4096); }

hipError_t launch_stats_partial(int dtype, const void *x, int64_t ldc, int64_t m, int C, int mode,
                                const float *mean, const float *rstd, const void *dy, int64_t dy_ldc,
                                float *part, int64_t R, hipStream_t s, const float *ctr)
{
    // operands each mode reads: refuse a launch that would dereference NULL
    if (!x || !part || ((mode == ST_SQDEV || mode == ST_DYX) && !mean) || (mode == ST_DYX && (!rstd || !dy)))
        return hipErrorInvalidValue;
    const int cb = (int)ceil_div(C, stats_ch_per_block(dtype));
    const int64_t rpb = ceil_div(m, R);
    dim3 grid((unsigned)ceil_div(m, rpb), (unsigned)cb);
    const double es = dtype == DT_BF16 ? 2.0 : 4.0;
    TraceScope tr(KC_SWEEP, KID_STATS_SWEEP, s, (mode == ST_DYX ? 2.0 : 1.0) * (double)m * C * es, 0.0);
    auto go = [&](auto kern, auto tag) {
        using T = decltype(tag);
        hipLaunchKernelGGL(kern, grid, dim3(kThreads), 0, s, (const T *)x, ldc, m, C, mean, rstd, (const T *)dy,
                           dy_ldc, rpb, part, ctr);
    };
    if (dtype == DT_BF16) {
        switch (mode) {
        case ST_SUMSQ: go(k_stats_partial<bf16_t, ST_SUMSQ>, bf16_t()); break;
        case ST_SUM: go(k_stats_partial<bf16_t, ST_SUM>, bf16_t()); break;
        case ST_SQDEV: go(k_stats_partial<bf16_t, ST_SQDEV>, bf16_t()); break;
        default: go(k_stats_partial<bf16_t, ST_DYX>, bf16_t()); break;
        }
    } else {
        switch (mode) {
        case ST_SUMSQ: go(k_stats_partial<float, ST_SUMSQ>, float()); break;
        case ST_SUM: go(k_stats_partial<float, ST_SUM>, float()); break;
        case ST_SQDEV: go(k_stats_partial<float, ST_SQDEV>, float()); break;
        default: go(k_stats_partial<float, ST_DYX>, float()); break;
        }
    }
    return hipGetLastError();
}

int stats_combine_splits(int64_t R)
{
    int64_t rs = R / 64;
    return (int)(rs < 1 ? 1 : (rs > kRedMaxRS ? kRedMaxRS : rs));
}

hipError_t launch_stats_finalize(const float *part, int64_t R, int C, int64_t m, int mode, float eps, float *mean,
                                 float *var, float *rstd, float *dbeta, float *dgamma, void *red, hipStream_t s,
                                 const SplitTerms *split)
{
    if (!part || !red || (mode == FIN_MVF && (!mean || !rstd)) || (mode == FIN_MEAN && !mean) ||
        (mode == FIN_VAR && !rstd) || (mode == FIN_BWD && (!dbeta || !dgamma)))
        return hipErrorInvalidValue;
    SplitTerms st{nullptr, nullptr, nullptr, nullptr, 0, nullptr, nullptr, nullptr, 0.f, nullptr};
    if (split && split->alpha) {
        if (mode != FIN_BWD || !split->gamma || !split->rstd || !split->betap) return hipErrorInvalidValue;
        st = *split;
    }
    if (split && (split->shift || split->rmean || split->mean_lo)) {
        if ((split->shift && mode != FIN_MVF) || (split->mean_lo && mode != FIN_MVF && mode != FIN_MEAN) ||
            (split->rmean && mode != FIN_MVF && mode != FIN_VAR) ||
            (!split->rmean && split->rvar) || split->alpha || (mode == FIN_VAR && split->rmean && !mean))
            return hipErrorInvalidValue;
        st.shift = split->shift; st.rmean = split->rmean; st.rvar = split->rvar; st.momentum = split->momentum;
        st.mean_lo = split->mean_lo;
    }
    if (R <= kCombineOneMaxRows) {
        TraceScope tr(KC_SMALL, KID_COMBINE, s, (double)R * 2 * C * 4 + 3.0 * C * 4, 0.0);
        hipLaunchKernelGGL(k_stats_combine_one, dim3((unsigned)ceil_div(C, 8)), dim3(kThreads), 0, s, part, R, C, m,
                           mode, eps, mean, var, rstd, dbeta, dgamma, st);
        return hipGetLastError();
    }
    double *lvl1 = reinterpret_cast<double *>(red);
    const int RS = stats_combine_splits(R);
    {
        TraceScope tr(KC_SMALL, KID_COMBINE, s, (double)R * 2 * C * 4 + (double)RS * 2 * C * 8, 0.0);
        hipLaunchKernelGGL(k_stats_combine1, dim3((unsigned)ceil_div(C, 64), (unsigned)RS), dim3(kThreads), 0, s, part,
                           R, C, lvl1);
    }
    TraceScope tr(KC_SMALL, KID_COMBINE, s, (double)RS * 2 * C * 8 + 3.0 * C * 4, 0.0);
    hipLaunchKernelGGL(k_stats_combine2, dim3((unsigned)ceil_div(C, kThreads)), dim3(kThreads), 0, s, lvl1, RS, C, m,
                       mode, eps, mean, var, rstd, dbeta, dgamma, st);
    return hipGetLastError();
}

hipError_t launch_elementwise(int dtype, int mode, int64_t m, int C, const void *x, int64_t x_ldc, const void *x2,
                              int64_t x2_ldc, const float *gamma, const float *beta, const float *mean,
                              const float *rstd, const float *dgamma, const float *dbeta, void *out,
                              int64_t out_ldc, int accumulate, hipStream_t s, const float *ctr)
{
    const bool two = mode == EW_DX || mode == EW_RELUBWD || mode == EW_BNADDRELU || mode == EW_ADDRELU ||
                     mode == EW_SPLITDX;
    if (!x || !out || (two && !x2) || (mode == EW_DX && (!gamma || !rstd || !mean || !dgamma || !dbeta)) ||
        (mode == EW_SPLITDX && (!rstd || !mean || !dgamma || !dbeta)) ||
        ((mode == EW_APPLY || mode == EW_BNADDRELU) && (!gamma || !beta || !mean || !rstd)))
        return hipErrorInvalidValue;
    // eight rows per thread: two four-row batches in flight per thread
    const int cb = (int)ceil_div(C, stats_ch_per_block(dtype));
    const int vb = (int)(C / stats_vec(dtype) < kStatsMaxVec ? C / stats_vec(dtype) : kStatsMaxVec);
    const int64_t rpb = (int64_t)(kThreads / vb) * 8;
    dim3 grid((unsigned)ceil_div(m, rpb), (unsigned)cb);
    const double sweeps = mode == EW_DX || mode == EW_SPLITDX ? 3.0 + (accumulate ? 1.0 : 0.0) : (two ? 3.0 : 2.0);
    TraceScope tr(KC_SWEEP, KID_ELEMENTWISE, s, sweeps * (double)m * C * (dtype == DT_BF16 ? 2 : 4), 0.0);
    auto go = [&](auto kern, auto tag) {
        using T = decltype(tag);
        hipLaunchKernelGGL(kern, grid, dim3(kThreads), 0, s, m, C, (const T *)x, x_ldc, (const T *)x2, x2_ldc, gamma,
                           beta, mean, rstd, dgamma, dbeta, (T *)out, out_ldc, rpb, ctr);
    };
    if (dtype == DT_BF16) {
        if (mode == EW_DX) {
            if (accumulate) go(k_elementwise<bf16_t, EW_DX, true>, bf16_t());
            else go(k_elementwise<bf16_t, EW_DX, false>, bf16_t());
        } else if (mode == EW_SPLITDX) {
            if (accumulate) go(k_elementwise<bf16_t, EW_SPLITDX, true>, bf16_t());
            else go(k_elementwise<bf16_t, EW_SPLITDX, false>, bf16_t());
        } else if (mode == EW_APPLY) go(k_elementwise<bf16_t, EW_APPLY, false>, bf16_t());
        else if (mode == EW_RELU) go(k_elementwise<bf16_t, EW_RELU, false>, bf16_t());
        else if (mode == EW_BNADDRELU) go(k_elementwise<bf16_t, EW_BNADDRELU, false>, bf16_t());
        else if (mode == EW_ADDRELU) go(k_elementwise<bf16_t, EW_ADDRELU, false>, bf16_t());
        else go(k_elementwise<bf16_t, EW_RELUBWD, false>, bf16_t());
    } else {
        if (mode == EW_DX) {
            if (accumulate) go(k_elementwise<float, EW_DX, true>, float());
            else go(k_elementwise<float, EW_DX, false>, float());
        } else if (mode == EW_SPLITDX) {
            if (accumulate) go(k_elementwise<float, EW_SPLITDX, true>, float());
            else go(k_elementwise<float, EW_SPLITDX, false>, float());
        } else if (mode == EW_APPLY) go(k_elementwise<float, EW_APPLY, false>, float());
        else if (mode == EW_RELU) go(k_elementwise<float, EW_RELU, false>, float());
        else if (mode == EW_BNADDRELU) go(k_elementwise<float, EW_BNADDRELU, false>, float());
        else if (mode == EW_ADDRELU) go(k_elementwise<float, EW_ADDRELU, false>, float());
        else go(k_elementwise<float, EW_RELUBWD, false>, float());
    }
    return hipGetLastError();
}

hipError_t launch_addrelu_bwd(int dtype, int64_t m, int C, const void *g, int64_t g_ldc, const void *out,
                              int64_t out_ldc, const void *y, int64_t y_ldc, const float *mean, const float *rstd,
                              void *gm, int64_t gm_ldc, float *part, int64_t R, hipStream_t s, const float *ctr)
{
    if (!g || !out || !y || !mean || !rstd || !gm || !part) return hipErrorInvalidValue;
    const int cb = (int)ceil_div(C, stats_ch_per_block(dtype));
    const int64_t rpb = ceil_div(m, R);
    dim3 grid((unsigned)ceil_div(m, rpb), (unsigned)cb);
    TraceScope tr(KC_SWEEP, KID_ELEMENTWISE, s, 4.0 * (double)m * C * (dtype == DT_BF16 ? 2 : 4), 0.0);
    if (dtype == DT_BF16)
        hipLaunchKernelGGL(k_addrelu_bwd<bf16_t>, grid, dim3(kThreads), 0, s, (const bf16_t *)g, g_ldc,
                           (const bf16_t *)out, out_ldc, (const bf16_t *)y, y_ldc, m, C, mean, rstd, (bf16_t *)gm,
                           gm_ldc, rpb, part, ctr);
    else
        hipLaunchKernelGGL(k_addrelu_bwd<float>, grid, dim3(kThreads), 0, s, (const float *)g, g_ldc,
                           (const float *)out, out_ldc, (const float *)y, y_ldc, m, C, mean, rstd, (float *)gm, gm_ldc,
                           rpb, part, ctr);
    return hipGetLastError();
}

hipError_t launch_avgpool2(int dtype, int n, int h, int w, int C, const void *x, int64_t ldc, void *y, int64_t y_ldc,
                           hipStream_t s)
{
    const int64_t total = (int64_t)n * (h / 2) * (w / 2) * (C / (dtype == DT_BF16 ? 8 : 4));
    const int grid = grid_cap(ceil_div(total, kThreads));
    TraceScope tr(KC_SWEEP, KID_POOL, s, 1.25 * (double)n * h * w * C * (dtype == DT_BF16 ? 2 : 4), 0.0);
    if (dtype == DT_BF16)
        hipLaunchKernelGGL(k_avgpool2<bf16_t>, dim3(grid), dim3(kThreads), 0, s, n, h, w, C, (const bf16_t *)x, ldc,
                           (bf16_t *)y, y_ldc);
    else
        hipLaunchKernelGGL(k_avgpool2<float>, dim3(grid), dim3(kThreads), 0, s, n, h, w, C, (const float *)x, ldc,
                           (float *)y, y_ldc);
    return hipGetLastError();
}

hipError_t launch_avgpool2_bwd(int dtype, int n, int h, int w, int C, const void *g, int64_t g_ldc, void *gx,
                               int64_t ldc, hipStream_t s)
{
    const int64_t total = (int64_t)n * h * w * (C / (dtype == DT_BF16 ? 8 : 4));
    const int grid = grid_cap(ceil_div(total, kThreads));
    TraceScope tr(KC_SWEEP, KID_POOL, s, 1.25 * (double)n * h * w * C * (dtype == DT_BF16 ? 2 : 4), 0.0);
    if (dtype == DT_BF16)
        hipLaunchKernelGGL(k_avgpool2_bwd<bf16_t>, dim3(grid), dim3(kThreads), 0, s, n, h, w, C, (const bf16_t *)g,
                           g_ldc, (bf16_t *)gx, ldc);
    else
        hipLaunchKernelGGL(k_avgpool2_bwd<float>, dim3(grid), dim3(kThreads), 0, s, n, h, w, C, (const float *)g,
                           g_ldc, (float *)gx, ldc);
    return hipGetLastError();
}

hipError_t launch_copy16(const void *src, void *dst, int64_t nvec, hipStream_t s)
{
    TraceScope tr(KC_SWEEP, KID_COPY, s, 32.0 * (double)nvec, 0.0);
    const int64_t per = ceil_div(nvec, 4096) < kThreads ? kThreads : ceil_div(nvec, 4096);
    hipLaunchKernelGGL(k_copy16, dim3((unsigned)ceil_div(nvec, per)), dim3(kThreads), 0, s, (const vec16 *)src,
                       (vec16 *)dst, nvec, per);
    return hipGetLastError();
}

hipError_t launch_bwd_tail(const float *wpart, int64_t S, int64_t len, float *dw, const float *spart, int64_t R,
                           int C, int64_t m, float *dbeta, float *dgamma, const SplitTerms *split, hipStream_t s)
{
    if (!wpart || !dw || (len % 4) || S < 1 || !spart || !dbeta || !dgamma || R > kCombineOneMaxRows)
        return hipErrorInvalidValue;
    SplitTerms st{nullptr, nullptr, nullptr, nullptr, 0};
    if (split && split->alpha) {
        if (!split->gamma || !split->rstd || !split->betap) return hipErrorInvalidValue;
        st = *split;
    }
    const int nb_sum = (int)ceil_div(len / 4, kTailF4);
    const int nb_comb = (int)ceil_div(C, 8);
    TraceScope tr(KC_SMALL, KID_SPLITK_SUM, s, 4.0 * (double)len * (S + 1) + (double)R * 2 * C * 4, 0.0);
    hipLaunchKernelGGL(k_bwd_tail, dim3((unsigned)(nb_sum + nb_comb)), dim3(kThreads), 0, s, wpart, S, len, dw, nb_sum,
                       spart, R, C, m, dbeta, dgamma, st);
    return hipGetLastError();
}

int sum_partials_groups(int64_t S) { return (int)(S < 8 ? S : 8); }

hipError_t launch_sum_partials(const float *part, int64_t S, int64_t len, float *out, void *red, hipStream_t s)
{
    const int SG = sum_partials_groups(S);
    if (!part || !out || (len % 4) || (SG > 1 && !red)) return hipErrorInvalidValue;
    const unsigned gx = (unsigned)ceil_div(len, 4 * kThreads);
    float *lvl1 = SG > 1 ? reinterpret_cast<float *>(red) : out;
    {
        TraceScope tr(KC_SMALL, KID_SPLITK_SUM, s, 4.0 * (double)len * (S + SG), 0.0);
        hipLaunchKernelGGL(k_sum_partials1, dim3(gx, (unsigned)SG), dim3(kThreads), 0, s, part, S, len, lvl1);
    }
    if (SG > 1) {
        TraceScope tr(KC_SMALL, KID_SPLITK_SUM, s, 4.0 * (double)len * (SG + 1), 0.0);
        hipLaunchKernelGGL(k_sum_partials2, dim3(gx), dim3(kThreads), 0, s, lvl1, SG, len, out);
    }
    return hipGetLastError();
}

}  // namespace bnr
