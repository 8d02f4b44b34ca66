// conv1x1.hip -- persistent 1x1 CONV (forward and data gradient) on the
// gfx950 matrix cores with the BN fission/fusion prologues and epilogues.
//
// One workgroup per CU (512 threads, 8 waves) keeps the whole weight matrix
// in LDS -- read once from its [c_in][c_out] layout, transposed on load for
// the forward GEMM -- and walks 128-pixel tiles t, t+G, t+2G, ...  For each
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
constexpr int kP1NV = 8;        // 16-byte vectors per thread for a tile operand

struct P1Geom {
    int KP, NP, lda, ldw, ldc;
    size_t region, lds;
};

template <typename T>
static P1Geom p1_geom(int K, int N)
{
    const int PAD = 16 / (int)sizeof(T);
    P1Geom g;
    g.KP = (int)((K + 31) / 32 * 32);
    g.NP = N <= 32 ? 32 : (N <= 64 ? 64 : (N <= 128 ? 128 : 256));
    g.lda = g.KP + PAD;
    g.ldw = g.KP + PAD;
    g.ldc = g.NP + PAD;
    const size_t a = (size_t)kP1BM * g.lda, c = (size_t)kP1BM * g.ldc;
    const size_t red = (size_t)2 * (kP1Threads / (g.NP / (16 / sizeof(T)))) * g.NP * sizeof(float) / sizeof(T);
    g.region = a > c ? (a > red ? a : red) : (c > red ? c : red);
    g.lds = ((size_t)g.NP * g.ldw + g.region) * sizeof(T) + (size_t)(5 * g.KP + 4 * g.NP) * sizeof(float);
    return g;
}

// NVA: upper bound of 16-byte A vectors per thread and tile (compile time, so
// the operand registers stay in VGPRs); IO: 0 = A only, 1 = A + epilogue
// operand, 2 = A + second prologue operand (PRO_BNGRAD) + epilogue operand.
template <typename T, int CBW, int NVA, int IO, int BM>
__global__ __launch_bounds__(kP1Threads) void k_conv1x1(RowsParams p, P1Geom g, int ntiles)
{
    using M = Mfma<T>;
    constexpr int VEC = Elem<T>::VEC;
    constexpr int RPT0 = BM * (32 * CBW / VEC) / kP1Threads;
    constexpr int RPT = RPT0 > 0 ? RPT0 : 1;                     // epilogue rows per thread
    constexpr int RB = BM / 64;                                  // 16-row MFMA blocks per wave
    constexpr int NVB = IO == 2 ? NVA : 1, NVX = IO >= 1 ? RPT : 1;
    extern __shared__ __align__(16) unsigned char smem[];
    T *Ws = reinterpret_cast<T *>(smem);
    T *As = Ws + (size_t)g.NP * g.ldw;
    T *Cs = As;                                           // output staging reuses the A tile
    float *coef = reinterpret_cast<float *>(As + g.region);
    float *epi = coef + 5 * g.KP;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;              // 4 x 2 waves: 32 rows x NP/2 columns each
    const int K = p.K, N = p.N, KP = g.KP, NP = g.NP;
    const int64_t m = p.m;
    const int H = p.h, W = p.w;
    const T *asrc = reinterpret_cast<const T *>(p.a);
    const T *asrc2 = reinterpret_cast<const T *>(p.a2);
    const T *wsrc = reinterpret_cast<const T *>(p.wraw);

    // ---- weights -> LDS as Ws[n][k] (zero outside K x N) ----
    if (!p.wtrans) {      // forward: W[k][n] (k = c_in, n = c_out); read rows of n, scatter to columns
        for (int i = tid; i < KP * (NP / VEC); i += kP1Threads) {
            const int k = i / (NP / VEC), n0 = (i % (NP / VEC)) * VEC;
            float f[VEC];
            if (k < K && n0 < N) Elem<T>::unpack(ldg16(wsrc + (int64_t)k * N + n0), f);
            else for (int e = 0; e < VEC; e++) f[e] = 0.f;
            #pragma unroll
            for (int e = 0; e < VEC; e++) Ws[(n0 + e) * g.ldw + k] = to_store<T>(f[e]);
        }
    } else {              // data gradient: W[n][k] (n = c_in, k = c_out): rows copy straight
        for (int i = tid; i < NP * (KP / VEC); i += kP1Threads) {
            const int n = i / (KP / VEC), k0 = (i % (KP / VEC)) * VEC;
            const vec16 v = (n < N && k0 < K) ? ldg16(wsrc + (int64_t)n * K + k0) : zero16();
            *reinterpret_cast<vec16 *>(Ws + n * g.ldw + k0) = v;
        }
    }
    // ---- per-channel prologue / epilogue parameters ----
    for (int c = tid; c < KP; c += kP1Threads) {
        float c0 = 0.f, c1 = 0.f, c2 = 0.f, c3 = 0.f, c4 = 0.f;
        if (c < K && p.pro == PRO_BNRELU) {
            c0 = p.p_mean[c]; c1 = p.p_gamma[c] * p.p_rstd[c]; c2 = p.p_beta[c];
        } else if (c < K && p.pro == PRO_BNGRAD) {
            const float inv_m = 1.0f / (float)m;
            c0 = p.p_mean[c]; c1 = p.p_rstd[c]; c2 = p.p_gamma[c] * p.p_rstd[c];
            c3 = p.p_dbeta[c] * inv_m; c4 = p.p_dgamma[c] * inv_m;
        }
        coef[c] = c0; coef[KP + c] = c1; coef[2 * KP + c] = c2; coef[3 * KP + c] = c3; coef[4 * KP + c] = c4;
    }
    for (int c = tid; c < NP; c += kP1Threads) {
        float e0 = 0.f, e1 = 1.f, e2 = 0.f, e3 = 0.f;
        if (c < N && p.epi == EPI_BNBWD) { e0 = p.e_mean[c]; e1 = p.e_rstd[c]; e2 = p.e_gamma[c]; e3 = p.e_beta[c]; }
        epi[c] = e0; epi[NP + c] = e1; epi[2 * NP + c] = e2; epi[3 * NP + c] = e3;
    }

    // ---- tile operand registers ----
    const int VPR = KP / VEC;                          // A vectors per row
    const int nva = (BM * VPR + kP1Threads - 1) / kP1Threads;
    // A slot j of this thread: 4 consecutive lanes cover 4 channel vectors (64
    // contiguous bytes of one pixel row), 16 lane groups cover 16 rows, so a
    // wave touches only 4 distinct prologue-coefficient addresses (LDS
    // broadcast, no bank conflicts).
    auto a_slot = [&](int j, int &r, int &c) __attribute__((always_inline)) {
        const int i = tid + j * kP1Threads;
        const int q = i >> 2;
        r = q % BM;
        c = ((q / BM) * 4 + (i & 3)) * VEC;
    };
    vec16 ra[NVA], rb[NVB];
    const bool pool = p.pro == PRO_POOLUP;
    auto load_a = [&](int tile) __attribute__((always_inline)) {
        const int64_t p0 = (int64_t)tile * BM;
        #pragma unroll
        for (int j = 0; j < NVA; j++) {
            int r, c;
            a_slot(j, r, c);
            const int64_t pp = p0 + r;
            const bool ok = j < nva && c < K && pp < m;
            int64_t q = pp;
            if (pool) {
                const int64_t img = pp / ((int64_t)H * W);
                const int rem = (int)(pp - img * H * W);
                const int y = rem / W, x = rem - y * W;
                q = (img * (H / 2) + y / 2) * (W / 2) + x / 2;
            }
            const vec16 va = ok ? ldg16(asrc + q * p.a_ldc + c) : zero16();
            ra[j] = va;
            if (IO == 2) rb[j < NVB ? j : 0] = ok ? ldg16(asrc2 + pp * p.a2_ldc + c) : zero16();
        }
    };
    auto store_a = [&](int tile) __attribute__((always_inline)) {
        const int64_t p0 = (int64_t)tile * BM;
        #pragma unroll
        for (int j = 0; j < NVA; j++) {
            if (j >= nva) continue;
            int r, c;
            a_slot(j, r, c);
            if (c >= KP) continue;
            const bool valid = p0 + r < m && c < K;
            vec16 out = ra[j];
            if (p.pro != PRO_NONE) {
                float f[VEC];
                Elem<T>::unpack(ra[j], f);
                if (p.pro == PRO_BNRELU) {
                    #pragma unroll
                    for (int e = 0; e < VEC; e++) {
                        const float t = (f[e] - coef[c + e]) * coef[KP + c + e] + coef[2 * KP + c + e];
                        f[e] = valid && t > 0.f ? t : 0.f;
                    }
                } else if (p.pro == PRO_RELU) {
                    #pragma unroll
                    for (int e = 0; e < VEC; e++) f[e] = f[e] > 0.f ? f[e] : 0.f;
                } else if (IO == 2 && p.pro == PRO_BNGRAD) {
                    float x[VEC];
                    Elem<T>::unpack(rb[j < NVB ? j : 0], x);
                    #pragma unroll
                    for (int e = 0; e < VEC; e++) {
                        const float xh = (x[e] - coef[c + e]) * coef[KP + c + e];
                        const float d = coef[2 * KP + c + e] * (f[e] - coef[3 * KP + c + e] - xh * coef[4 * KP + c + e]);
                        f[e] = valid ? d : 0.f;
                    }
                } else {  // PRO_POOLUP
                    #pragma unroll
                    for (int e = 0; e < VEC; e++) f[e] *= 0.25f;
                }
                out = Elem<T>::pack(f);
            }
            *reinterpret_cast<vec16 *>(As + r * g.lda + c) = out;
        }
    };

    // ---- epilogue mapping: thread = one channel vector of rows r0, r0+RSTEP, ... ----
    const int VPRO = NP / VEC, RSTEP = kP1Threads / VPRO;
    const int v = tid % VPRO, r0 = tid / VPRO;
    const int n = v * VEC;
    const bool col_ok = n < N;
    vec16 rx[NVX];
    float s1[VEC], s2[VEC];
    #pragma unroll
    for (int e = 0; e < VEC; e++) { s1[e] = 0.f; s2[e] = 0.f; }
    T *yout = reinterpret_cast<T *>(p.y);
    const T *exs = reinterpret_cast<const T *>(p.ex);
    const bool epi_reads = p.epi == EPI_BNBWD || p.epi == EPI_RELUMASK || (p.epi == EPI_STORE && p.accumulate);
    auto load_epi = [&](int tile) __attribute__((always_inline)) {
        const int64_t p0 = (int64_t)tile * BM;
        if (IO == 0) return;
        #pragma unroll
        for (int j = 0; j < NVX; j++) {
            rx[j] = zero16();
            if (!epi_reads || !col_ok) continue;
            const int64_t pp = p0 + r0 + j * RSTEP;
            if (r0 + j * RSTEP >= BM || pp >= m) continue;
            rx[j] = p.epi == EPI_STORE ? ldg16(yout + pp * p.y_ldc + n) : ldg16(exs + pp * p.ex_ldc + n);
        }
    };

    __syncthreads();
    // this thread's epilogue channels are fixed: keep their BN parameters in registers
    float eM[VEC], eR[VEC], eG[VEC], eB[VEC];
    #pragma unroll
    for (int e = 0; e < VEC; e++) {
        eM[e] = epi[n + e]; eR[e] = epi[NP + n + e]; eG[e] = epi[2 * NP + n + e]; eB[e] = epi[3 * NP + n + e];
    }
    int tile = blockIdx.x;
    if (tile < ntiles) load_a(tile);
    for (; tile < ntiles; tile += gridDim.x) {
        store_a(tile);
        __syncthreads();
        if (tile + (int)gridDim.x < ntiles) load_a(tile + gridDim.x);
        load_epi(tile);
        // ---- matrix cores: 32 rows x NP/2 columns per wave ----
        f32x4 acc[RB][CBW];
        #pragma unroll
        for (int ib = 0; ib < RB; ib++)
            #pragma unroll
            for (int cb = 0; cb < CBW; cb++) acc[ib][cb] = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int k0 = 0; k0 < KP; k0 += M::KSTEP) {
            const int kofs = k0 + (lane >> 4) * M::KPL;
            typename M::frag a[RB];
            #pragma unroll
            for (int ib = 0; ib < RB; ib++) a[ib] = M::load(As + (wm * (16 * RB) + ib * 16 + (lane & 15)) * g.lda + kofs);
            #pragma unroll
            for (int cb = 0; cb < CBW; cb++) {
                const typename M::frag b = M::load(Ws + (wn * (NP / 2) + cb * 16 + (lane & 15)) * g.ldw + kofs);
                #pragma unroll
                for (int ib = 0; ib < RB; ib++) M::mma(acc[ib][cb], a[ib], b);
            }
        }
        __syncthreads();
        #pragma unroll
        for (int ib = 0; ib < RB; ib++)
            #pragma unroll
            for (int cb = 0; cb < CBW; cb++)
                #pragma unroll
                for (int i = 0; i < 4; i++) {
                    const int row = wm * (16 * RB) + ib * 16 + (lane >> 4) * 4 + i;
                    const int col = wn * (NP / 2) + cb * 16 + (lane & 15);
                    Cs[row * g.ldc + col] = to_store<T>(acc[ib][cb][i]);
                }
        __syncthreads();
        // ---- epilogue row pass ----
        const int64_t p0 = (int64_t)tile * BM;
        if (col_ok) {
            #pragma unroll
            for (int j = 0; j < RPT; j++) {
                const int r = r0 + j * RSTEP;
                const int64_t pp = p0 + r;
                if (r >= BM || pp >= m) continue;
                const vec16 cv = *reinterpret_cast<const vec16 *>(Cs + r * g.ldc + n);
                T *dst = yout + pp * p.y_ldc + n;
                float f[VEC];
                Elem<T>::unpack(cv, f);
                if (p.epi == EPI_STORE) {
                    if (IO >= 1 && p.accumulate) {
                        float old[VEC];
                        Elem<T>::unpack(rx[j < NVX ? j : 0], old);
                        #pragma unroll
                        for (int e = 0; e < VEC; e++) f[e] += old[e];
                        stg16(dst, Elem<T>::pack(f));
                    } else {
                        stg16(dst, cv);
                    }
                } else if (p.epi == EPI_STATS) {
                    stg16(dst, cv);
                    #pragma unroll
                    for (int e = 0; e < VEC; e++) { s1[e] += f[e]; s2[e] += f[e] * f[e]; }
                } else if (IO >= 1 && p.epi == EPI_RELUMASK) {
                    float yv[VEC];
                    Elem<T>::unpack(rx[j < NVX ? j : 0], yv);
                    #pragma unroll
                    for (int e = 0; e < VEC; e++) f[e] = yv[e] > 0.f ? f[e] : 0.f;
                    stg16(dst, Elem<T>::pack(f));
                } else if (IO >= 1) {  // EPI_BNBWD
                    float x[VEC];
                    Elem<T>::unpack(rx[j < NVX ? j : 0], x);
                    #pragma unroll
                    for (int e = 0; e < VEC; e++) {
                        const float xh = (x[e] - eM[e]) * eR[e];
                        const float yv = eG[e] * xh + eB[e];
                        const float d = yv > 0.f ? f[e] : 0.f;
                        f[e] = d;
                        s1[e] += d;
                        s2[e] += d * xh;
                    }
                    stg16(dst, Elem<T>::pack(f));
                }
            }
        }
        __syncthreads();
    }

    // ---- per-workgroup statistics partial row ----
    if (p.epi == EPI_STATS || p.epi == EPI_BNBWD) {
        float *red = reinterpret_cast<float *>(As);
        #pragma unroll
        for (int e = 0; e < VEC; e++) {
            red[r0 * NP + n + e] = s1[e];
            red[(RSTEP + r0) * NP + n + e] = s2[e];
        }
        __syncthreads();
        for (int c = tid; c < N; c += kP1Threads) {
            float a = 0.f, b = 0.f;
            for (int j = 0; j < RSTEP; j++) { a += red[j * NP + c]; b += red[(RSTEP + j) * NP + c]; }
            p.part[(int64_t)blockIdx.x * 2 * N + c] = a;
            p.part[(int64_t)blockIdx.x * 2 * N + N + c] = b;
        }
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

bool conv1x1_supported(int dtype, int K, int N)
{
    if (K > 256 || N > 256 || (dtype != DT_BF16 && N > 128)) return false;
    const P1Geom g = dtype == DT_BF16 ? p1_geom<bf16_t>(K, N) : p1_geom<float>(K, N);
    if (g.lds > 150 * 1024) return false;
    const int VEC = dtype == DT_BF16 ? 8 : 4;
    if ((int64_t)kP1BM * (g.KP / VEC) > (int64_t)kP1NV * kP1Threads) return false;      // A tile registers
    if (kP1BM / (kP1Threads / (g.NP / VEC)) > kP1NV) return false;                       // epilogue registers
    return true;
}

int64_t conv1x1_partial_rows(int64_t m)
{
    const int64_t tiles = ceil_div(m, kP1BM);
    const int64_t g = device_cus();
    return tiles < g ? tiles : g;
}

template <typename T, int CBW, int NVA, int IO, int BM>
static hipError_t run_p1(const RowsParams &p, const P1Geom &g, hipStream_t s)
{
    auto kern = k_conv1x1<T, CBW, NVA, IO, BM>;
    static bool attr_set = false;
    if (!attr_set) {
        const hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    const int ntiles = (int)ceil_div(p.m, BM);
    const int grid = (int)conv1x1_partial_rows(p.m);
    const double e = sizeof(T), m = (double)p.m;
    double a = m * p.K;
    if (p.pro == PRO_BNGRAD) a *= 2.0;
    if (p.pro == PRO_POOLUP) a /= 4.0;
    double out = m * p.N;
    if (p.epi == EPI_BNBWD || p.epi == EPI_RELUMASK || (p.epi == EPI_STORE && p.accumulate)) out += m * p.N;
    TraceScope tr(KC_CONV, KID_CONV_1X1, s, e * (a + out + (double)p.K * p.N), 2.0 * m * p.K * p.N);
    hipLaunchKernelGGL(kern, dim3(grid), dim3(kP1Threads), g.lds, s, p, g, ntiles);
    return hipGetLastError();
}

// Tile height: 128 rows unless the operand registers of the variant would not
// fit the 256 VGPRs a wave has at two waves per SIMD; then 64 rows, which
// halves every per-thread operand array.
template <typename T, int CBW, int NVA128, int IO>
static hipError_t run_p1_bm(const RowsParams &p, const P1Geom &g, hipStream_t s)
{
    constexpr bool small = (CBW == 8 && IO >= 1) || (NVA128 == 8 && IO == 2);
    if constexpr (small) return run_p1<T, CBW, 4, IO, 64>(p, g, s);
    else return run_p1<T, CBW, NVA128, IO, 128>(p, g, s);
}

template <typename T, int NVA128, int IO>
static hipError_t run_p1_cbw(const RowsParams &p, const P1Geom &g, hipStream_t s)
{
    switch (g.NP / 32) {
    case 1: return run_p1_bm<T, 1, NVA128, IO>(p, g, s);
    case 2: return run_p1_bm<T, 2, NVA128, IO>(p, g, s);
    case 4: return run_p1_bm<T, 4, NVA128, IO>(p, g, s);
    default:
        if constexpr (sizeof(T) == 2) return run_p1_bm<T, 8, NVA128, IO>(p, g, s);
        else return hipErrorInvalidValue;      // float with 256 output columns exceeds LDS
    }
}

template <typename T>
static hipError_t run_p1_io(const RowsParams &p, const P1Geom &g, int io, hipStream_t s)
{
    const int nva = (int)ceil_div((int64_t)kP1BM * (g.KP / Elem<T>::VEC), kP1Threads);
    if (nva <= 4) {
        if (io == 0) return run_p1_cbw<T, 4, 0>(p, g, s);
        if (io == 1) return run_p1_cbw<T, 4, 1>(p, g, s);
        return run_p1_cbw<T, 4, 2>(p, g, s);
    }
    if (io == 0) return run_p1_cbw<T, 8, 0>(p, g, s);
    if (io == 1) return run_p1_cbw<T, 8, 1>(p, g, s);
    return run_p1_cbw<T, 8, 2>(p, g, s);
}

hipError_t launch_conv1x1(const RowsParams &p, hipStream_t s)
{
    if (!p.a || !p.wraw || !p.y || p.taps != 1 || !conv1x1_supported(p.dtype, p.K, p.N)) return hipErrorInvalidValue;
    if (p.pro == PRO_BNRELU && (!p.p_mean || !p.p_gamma || !p.p_rstd || !p.p_beta)) return hipErrorInvalidValue;
    if (p.pro == PRO_BNGRAD && (!p.a2 || !p.p_mean || !p.p_rstd || !p.p_gamma || !p.p_dbeta || !p.p_dgamma))
        return hipErrorInvalidValue;
    if ((p.epi == EPI_STATS || p.epi == EPI_BNBWD) && !p.part) return hipErrorInvalidValue;
    if (p.epi == EPI_BNBWD && (!p.ex || !p.e_mean || !p.e_rstd || !p.e_gamma || !p.e_beta)) return hipErrorInvalidValue;
    if (p.epi == EPI_RELUMASK && !p.ex) return hipErrorInvalidValue;
    const bool epi_reads = p.epi == EPI_BNBWD || p.epi == EPI_RELUMASK || (p.epi == EPI_STORE && p.accumulate);
    const int io = p.pro == PRO_BNGRAD ? 2 : (epi_reads ? 1 : 0);
    if (p.dtype == DT_BF16) return run_p1_io<bf16_t>(p, p1_geom<bf16_t>(p.K, p.N), io, s);
    return run_p1_io<float>(p, p1_geom<float>(p.K, p.N), io, s);
}

}  // namespace bnr
