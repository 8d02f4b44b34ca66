// conv3x3.hip -- persistent 3x3 CONV (stride 1, zero padding 1), forward and
// data gradient, on the gfx950 matrix cores with the BN fission/fusion
// prologues and epilogues.
//
// One 512-thread workgroup per CU owns a contiguous range of pixel rows
// [P0, P1) of the NHWC tensor (pixel = row of the GEMM) and keeps
//   * the weights of all nine taps in LDS, read once from [kh][kw][ci][co]
//     (transposed on load for the forward GEMM, taps flipped for the data
//     gradient), and
//   * a ring buffer of input rows: a 128-row output tile at p0 needs the rows
//     [p0 - (W+1), p0 + 128 + W + 1); consecutive tiles share all but 128 of
//     them, so each input row is read from HBM and transformed by the
//     prologue once (no halo re-reads inside a workgroup).
// The 128 new rows of the next tile are loaded into registers while the
// matrix cores work on the current tile, together with the epilogue operand
// of the current tile.  Two waves per SIMD let one wave's prologue / epilogue
// arithmetic overlap the other's matrix-core work.  Taps that fall outside
// the image read a zero row of LDS: zero padding applies to the CONV input,
// i.e. after BN and ReLU.
//
// The epilogue stages the output tile through LDS so that every global access
// is a 16-byte vector of one pixel row, and keeps the per-channel statistics
// of the workgroup's rows in registers: one partial row per workgroup.
// Prologue / epilogue modes are those of conv_rows.hip.
#include "common.hpp"
#include "kernels.hpp"
#include "mfma.hpp"
#include "tiles.hpp"
#include "trace.hpp"

namespace bnr {

constexpr int kP3Threads = 512;
constexpr int kP3BM = 128;          // output rows per tile
constexpr int kP3MaxW = 62;         // widest image row (ring = 128 + 2 (W + 1) rows)

struct P3Geom {
    int KP, NP, lda, ldw, ldc, ring;
    size_t ring_bytes;              // ring rows + one zero row (also the final statistics scratch)
    size_t lds;
};

template <typename T>
static P3Geom p3_geom(int K, int N, int W)
{
    const int PAD = 16 / (int)sizeof(T);
    P3Geom g;
    g.KP = (K + 31) / 32 * 32;
    g.NP = N <= 32 ? 32 : (N <= 64 ? 64 : 128);
    g.lda = g.KP + PAD;
    g.ldw = g.KP + PAD;
    g.ldc = g.NP + PAD;
    g.ring = kP3BM + 2 * (W + 1);
    const size_t red = (size_t)2 * (kP3Threads / (g.NP / (16 / sizeof(T)))) * g.NP * sizeof(float);
    g.ring_bytes = (size_t)(g.ring + 1) * g.lda * sizeof(T);
    if (red > g.ring_bytes) g.ring_bytes = red;
    g.lds = (size_t)9 * g.NP * g.ldw * sizeof(T) + g.ring_bytes + (size_t)kP3BM * g.ldc * sizeof(T) +
            (size_t)(5 * g.KP + 4 * g.NP) * sizeof(float);
    return g;
}

// NPC: output columns (32, 64 or 128); WM: waves along the 128 tile rows
// (8 or 4; the other 8 / WM waves split the columns).  The epilogue kind EK
// and whether the prologue reads a second operand (PRO_BNGRAD) are
// compile-time, so the epilogue is straight-line code and the compiler can
// keep the next tile's loads in flight while it waits for the epilogue
// operand (a runtime mode switch makes it wait for every outstanding load at
// each branch).
template <typename T, int NPC, int WM, int EK, bool BNG>
__global__ __launch_bounds__(kP3Threads) void k_conv3x3(RowsParams p, P3Geom g)
{
    using M = Mfma<T>;
    constexpr int VEC = Elem<T>::VEC;
    constexpr int WN = 8 / WM;
    constexpr int RB = kP3BM / (16 * WM);                        // 16-row blocks per wave
    constexpr int CBW = NPC / (16 * WN);                         // 16-column blocks per wave
    constexpr int VPRO = NPC / VEC, RSTEP = kP3Threads / VPRO;
    constexpr int RPT = kP3BM / RSTEP > 0 ? kP3BM / RSTEP : 1;   // epilogue rows per thread
    constexpr bool READS = EK == EK_STORE_ACC || EK == EK_RELUMASK || EK == EK_BNBWD;
    constexpr int NVA = kP3BM * (128 / VEC) / kP3Threads;       // up to 128 input channels
    constexpr int NVB = BNG ? NVA : 1, NVX = READS ? RPT : 1;
    static_assert(RB >= 1 && CBW >= 1, "wave layout");
    extern __shared__ __align__(16) unsigned char smem[];
    T *Ws = reinterpret_cast<T *>(smem);                         // [9][NP][ldw]
    T *ring = Ws + (size_t)9 * NPC * g.ldw;                      // [ring + 1][lda]; row `ring` is zero
    T *Cs = reinterpret_cast<T *>(reinterpret_cast<unsigned char *>(ring) + g.ring_bytes);   // [BM][ldc]
    float *coef = reinterpret_cast<float *>(Cs + (size_t)kP3BM * g.ldc);
    float *epi = coef + 5 * g.KP;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave % WM, wn = wave / WM;
    const int K = p.K, N = p.N, KP = g.KP, RING = g.ring;
    const int m = (int)p.m;                                      // launcher: m < 2^30
    const int H = p.h, W = p.w, H1 = W + 1;
    const int P0 = (int)((int64_t)blockIdx.x * m / gridDim.x), P1 = (int)((int64_t)(blockIdx.x + 1) * m / gridDim.x);
    const T *wsrc = reinterpret_cast<const T *>(p.wraw);
    constexpr uint32_t ES = sizeof(T);
    // operand views as raw buffers (launcher guarantees each spans < 2^31 bytes)
    const int a_ldc = (int)p.a_ldc, a2_ldc = (int)p.a2_ldc, y_ldc = (int)p.y_ldc, ex_ldc = (int)p.ex_ldc;
    const __amdgpu_buffer_rsrc_t abuf = buf_view(p.a, (uint32_t)(((int64_t)(m - 1) * a_ldc + K) * ES));
    const __amdgpu_buffer_rsrc_t a2buf = buf_view(BNG ? p.a2 : p.a, BNG ? (uint32_t)(((int64_t)(m - 1) * a2_ldc + K) * ES) : 0u);
    const __amdgpu_buffer_rsrc_t ybuf = buf_view(p.y, (uint32_t)(((int64_t)(m - 1) * y_ldc + N) * ES));
    const __amdgpu_buffer_rsrc_t xbuf = buf_view(p.ex ? p.ex : p.y,
                                                 p.ex ? (uint32_t)(((int64_t)(m - 1) * ex_ldc + N) * ES) : 0u);

    // ---- weights -> LDS as Ws[tap][n][k] (zero outside K x N) ----
    if (!p.wtrans) {      // forward: W[tap][k][n] (k = c_in, n = c_out); scatter columns
        for (int i = tid; i < 9 * KP * VPRO; i += kP3Threads) {
            const int tap = i / (KP * VPRO), rem = i % (KP * VPRO);
            const int k = rem / VPRO, n0 = (rem % VPRO) * VEC;
            float f[VEC];
            if (k < K && n0 < N) Elem<T>::unpack(ldg16(wsrc + ((int64_t)tap * K + k) * N + n0), f);
            else for (int e = 0; e < VEC; e++) f[e] = 0.f;
            #pragma unroll
            for (int e = 0; e < VEC; e++) Ws[(tap * NPC + n0 + e) * g.ldw + k] = to_store<T>(f[e]);
        }
    } else {              // data gradient: W[8 - tap][n][k] (n = c_in, k = c_out); rows copy straight
        const int VPK = KP / VEC;
        for (int i = tid; i < 9 * NPC * VPK; i += kP3Threads) {
            const int tap = i / (NPC * VPK), rem = i % (NPC * VPK);
            const int n = rem / VPK, k0 = (rem % VPK) * VEC;
            const vec16 v = (n < N && k0 < K) ? ldg16(wsrc + ((int64_t)(8 - tap) * N + n) * K + k0) : zero16();
            *reinterpret_cast<vec16 *>(Ws + (tap * NPC + n) * g.ldw + k0) = v;
        }
    }
    for (int i = tid; i < KP / VEC; i += kP3Threads)               // the zero row
        *reinterpret_cast<vec16 *>(ring + (size_t)RING * g.lda + i * VEC) = zero16();
    // ---- per-channel prologue / epilogue parameters ----
    //   BNRELU: z = max(x * c0 + c1, 0) with c0 = gamma*rstd, c1 = beta - mean*gamma*rstd
    //   BNGRAD: d = c2 * (dy - c3 - (x - c0) * c1 * c4)
    for (int c = tid; c < KP; c += kP3Threads) {
        float c0 = 0.f, c1 = 0.f, c2 = 0.f, c3 = 0.f, c4 = 0.f;
        if (c < K && p.pro == PRO_BNRELU) {
            c0 = p.p_gamma[c] * p.p_rstd[c]; c1 = p.p_beta[c] - p.p_mean[c] * c0;
        } else if (c < K && p.pro == PRO_BNGRAD) {
            const float inv_m = 1.0f / (float)m;
            c0 = p.p_mean[c]; c1 = p.p_rstd[c]; c2 = p.p_gamma[c] * p.p_rstd[c];
            c3 = p.p_dbeta[c] * inv_m; c4 = p.p_dgamma[c] * inv_m;
        }
        coef[c] = c0; coef[KP + c] = c1; coef[2 * KP + c] = c2; coef[3 * KP + c] = c3; coef[4 * KP + c] = c4;
    }
    for (int c = tid; c < NPC; c += kP3Threads) {
        float e0 = 0.f, e1 = 1.f, e2 = 0.f, e3 = 0.f;
        if (c < N && EK == EK_BNBWD) { e0 = p.e_mean[c]; e1 = p.e_rstd[c]; e2 = p.e_gamma[c]; e3 = p.e_beta[c]; }
        epi[c] = e0; epi[NPC + c] = e1; epi[2 * NPC + c] = e2; epi[3 * NPC + c] = e3;
    }

    // ---- input batches: up to 128 consecutive rows, loaded to registers ----
    // Slot j of this thread: 4 consecutive lanes cover 4 channel vectors of
    // one row, 16 lane groups 16 rows (4 distinct coefficient addresses per
    // wave: LDS broadcast).
    const int VPR = KP / VEC;
    const int nva = (kP3BM * VPR + kP3Threads - 1) / kP3Threads;
    int sr[NVA], sc[NVA];
    #pragma unroll
    for (int j = 0; j < NVA; j++) {
        const int i = tid + j * kP3Threads;
        const int q = i >> 2;
        sr[j] = q % kP3BM;
        sc[j] = ((q / kP3BM) * 4 + (i & 3)) * VEC;
    }
    vec16 ra[NVA], rb[NVB];
    auto load_rows = [&](int q0, int cnt) __attribute__((always_inline)) {
        #pragma unroll
        for (int j = 0; j < NVA; j++) {
            const int q = q0 + sr[j];
            const bool ok = j < nva && sc[j] < K && sr[j] < cnt && q >= 0 && q < m;
            ra[j] = bld16(abuf, ok ? (uint32_t)(q * a_ldc + sc[j]) * ES : kBufOff);
            if (BNG) rb[j < NVB ? j : 0] = bld16(a2buf, ok ? (uint32_t)(q * a2_ldc + sc[j]) * ES : kBufOff);
        }
    };
    auto store_rows = [&](int q0, int cnt, int slot0) __attribute__((always_inline)) {
        #pragma unroll
        for (int j = 0; j < NVA; j++) {
            const int r = sr[j], c = sc[j];
            if (j >= nva || c >= KP || r >= cnt) continue;
            const int q = q0 + r;
            const bool valid = q >= 0 && q < m && c < K;
            vec16 out = ra[j];
            if (p.pro != PRO_NONE) {
                float f[VEC];
                Elem<T>::unpack(ra[j], f);
                if (p.pro == PRO_BNRELU) {
                    #pragma unroll
                    for (int e = 0; e < VEC; e++) {
                        const float t = __builtin_fmaf(f[e], coef[c + e], coef[KP + c + e]);
                        f[e] = valid && t > 0.f ? t : 0.f;
                    }
                } else if (p.pro == PRO_RELU) {
                    #pragma unroll
                    for (int e = 0; e < VEC; e++) f[e] = f[e] > 0.f ? f[e] : 0.f;
                } else if (BNG && p.pro == PRO_BNGRAD) {
                    float x[VEC];
                    Elem<T>::unpack(rb[j < NVB ? j : 0], x);
                    #pragma unroll
                    for (int e = 0; e < VEC; e++) {
                        const float xh = (x[e] - coef[c + e]) * coef[KP + c + e];
                        const float d = coef[2 * KP + c + e] * (f[e] - coef[3 * KP + c + e] - xh * coef[4 * KP + c + e]);
                        f[e] = valid ? d : 0.f;
                    }
                }
                out = Elem<T>::pack(f);
            }
            int s = slot0 + r;
            if (s >= RING) s -= RING;
            *reinterpret_cast<vec16 *>(ring + s * g.lda + c) = out;
        }
    };

    // ---- epilogue mapping: thread = one channel vector of rows r0, r0+RSTEP, ... ----
    const int v = tid % VPRO, r0 = tid / VPRO;
    const int n = v * VEC;
    const bool col_ok = n < N;
    vec16 rx[NVX];
    float s1[VEC], s2[VEC];
    #pragma unroll
    for (int e = 0; e < VEC; e++) { s1[e] = 0.f; s2[e] = 0.f; }
    T *yout = reinterpret_cast<T *>(p.y);
    auto load_epi = [&](int p0, int nrows) __attribute__((always_inline)) {
        if (!READS) return;
        #pragma unroll
        for (int j = 0; j < NVX; j++) {
            const int r = r0 + j * RSTEP;
            const int pp = p0 + r;
            const bool ok = col_ok && r < nrows;
            if (EK == EK_STORE_ACC) rx[j] = bld16(ybuf, ok ? (uint32_t)(pp * y_ldc + n) * ES : kBufOff);
            else rx[j] = bld16(xbuf, ok ? (uint32_t)(pp * ex_ldc + n) * ES : kBufOff);
        }
    };

    __syncthreads();
    float eM[VEC], eR[VEC], eG[VEC], eB[VEC];
    #pragma unroll
    for (int e = 0; e < VEC; e++) {
        eM[e] = epi[n + e]; eR[e] = epi[NPC + n + e]; eG[e] = epi[2 * NPC + n + e]; eB[e] = epi[3 * NPC + n + e];
    }

    // ---- ring fill: rows [P0 - H1, P0 + H1) ----
    int L = P0 - H1;                // next input row to load; its ring slot is slotL
    int slotL = 0;
    while (L < P0 + H1) {
        const int cnt = P0 + H1 - L < kP3BM ? P0 + H1 - L : kP3BM;
        load_rows(L, cnt);
        store_rows(L, cnt, slotL);
        L += cnt;
        slotL += cnt;
        if (slotL >= RING) slotL -= RING;
    }
    // prefetch the batch of the first tile
    int cnt = P1 + H1 - L < kP3BM ? P1 + H1 - L : kP3BM;
    load_rows(L, cnt);
    int sb = H1;                    // ring slot of the first row of the current tile

    for (int p0 = P0; p0 < P1; p0 += kP3BM) {
        const int nrows = P1 - p0 < kP3BM ? P1 - p0 : kP3BM;
        store_rows(L, cnt, slotL);
        L += cnt;
        slotL += cnt;
        if (slotL >= RING) slotL -= RING;
        __syncthreads();
        // epilogue operand first: the epilogue waits for it while the next
        // tile's rows (issued after it) may still be in flight
        load_epi(p0, nrows);
        cnt = P1 + H1 - L < kP3BM ? P1 + H1 - L : kP3BM;
        if (cnt > 0) load_rows(L, cnt);

        // ---- matrix cores: (16 RB) rows x (16 CBW) columns per wave, nine taps ----
        int hh[RB], ww[RB], rw[RB];
        #pragma unroll
        for (int ib = 0; ib < RB; ib++) {
            rw[ib] = wm * 16 * RB + ib * 16 + (lane & 15);
            const int pp = p0 + rw[ib];
            ww[ib] = pp % W;
            hh[ib] = (pp / W) % H;
        }
        f32x4 acc[RB][CBW];
        #pragma unroll
        for (int ib = 0; ib < RB; ib++)
            #pragma unroll
            for (int cb = 0; cb < CBW; cb++) acc[ib][cb] = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int tap = 0; tap < 9; tap++) {
            const int dh = tap / 3 - 1, dw = tap % 3 - 1;
            const int off = dh * W + dw;
            const T *arow[RB];
            #pragma unroll
            for (int ib = 0; ib < RB; ib++) {
                int s = sb + rw[ib] + off;
                if (s < 0) s += RING;
                if (s >= RING) s -= RING;
                const bool ok = rw[ib] < nrows && (unsigned)(hh[ib] + dh) < (unsigned)H &&
                                (unsigned)(ww[ib] + dw) < (unsigned)W;
                arow[ib] = ring + (ok ? s : RING) * g.lda + (lane >> 4) * M::KPL;
            }
            const T *brow = Ws + (tap * NPC + wn * 16 * CBW + (lane & 15)) * g.ldw + (lane >> 4) * M::KPL;
            for (int k0 = 0; k0 < KP; k0 += M::KSTEP) {
                typename M::frag a[RB];
                #pragma unroll
                for (int ib = 0; ib < RB; ib++) a[ib] = M::load(arow[ib] + k0);
                #pragma unroll
                for (int cb = 0; cb < CBW; cb++) {
                    const typename M::frag b = M::load(brow + cb * 16 * g.ldw + k0);
                    #pragma unroll
                    for (int ib = 0; ib < RB; ib++) M::mma(acc[ib][cb], a[ib], b);
                }
            }
        }
        #pragma unroll
        for (int ib = 0; ib < RB; ib++)
            #pragma unroll
            for (int cb = 0; cb < CBW; cb++)
                #pragma unroll
                for (int i = 0; i < 4; i++) {
                    const int row = wm * 16 * RB + ib * 16 + (lane >> 4) * 4 + i;
                    const int col = wn * 16 * CBW + cb * 16 + (lane & 15);
                    Cs[row * g.ldc + col] = to_store<T>(acc[ib][cb][i]);
                }
        __syncthreads();
        // ---- epilogue row pass: all outputs of this thread first (no branch,
        // invalid rows contribute zeros), then the stores back to back ----
        {
            vec16 vo[RPT];
            #pragma unroll
            for (int j = 0; j < RPT; j++) {
                const int r = r0 + j * RSTEP;
                const bool ok = col_ok && r < nrows;
                const vec16 cv = *reinterpret_cast<const vec16 *>(Cs + (r < kP3BM ? r : 0) * g.ldc + n);
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
                        const float fv = ok ? f[e] : 0.f;
                        s1[e] += fv;
                        s2[e] += fv * fv;
                    }
                } else if (EK == EK_RELUMASK) {
                    float yv[VEC];
                    Elem<T>::unpack(rx[j < NVX ? j : 0], yv);
                    #pragma unroll
                    for (int e = 0; e < VEC; e++) f[e] = yv[e] > 0.f ? f[e] : 0.f;
                    vo[j] = Elem<T>::pack(f);
                } else if (EK == EK_BNBWD) {
                    float x[VEC];
                    Elem<T>::unpack(rx[j < NVX ? j : 0], x);
                    #pragma unroll
                    for (int e = 0; e < VEC; e++) {
                        const float xh = (x[e] - eM[e]) * eR[e];
                        const float yv = eG[e] * xh + eB[e];
                        const float d = ok && yv > 0.f ? f[e] : 0.f;
                        f[e] = d;
                        s1[e] += d;
                        s2[e] += d * xh;
                    }
                    vo[j] = Elem<T>::pack(f);
                }
            }
            #pragma unroll
            for (int j = 0; j < RPT; j++) {
                const int r = r0 + j * RSTEP;
                if (col_ok && r < nrows) stg16(yout + (int64_t)(p0 + r) * y_ldc + n, vo[j]);
            }
        }
        sb += kP3BM;
        if (sb >= RING) sb -= RING;
        __syncthreads();
    }

    // ---- per-workgroup statistics partial row ----
    if (EK == EK_STATS || EK == EK_BNBWD) {
        float *red = reinterpret_cast<float *>(ring);
        #pragma unroll
        for (int e = 0; e < VEC; e++) {
            red[r0 * NPC + n + e] = s1[e];
            red[(RSTEP + r0) * NPC + n + e] = s2[e];
        }
        __syncthreads();
        for (int c = tid; c < N; c += kP3Threads) {
            float a = 0.f, b = 0.f;
            for (int j = 0; j < RSTEP; j++) { a += red[j * NPC + c]; b += red[(RSTEP + j) * NPC + c]; }
            p.part[(int64_t)blockIdx.x * 2 * N + c] = a;
            p.part[(int64_t)blockIdx.x * 2 * N + N + c] = b;
        }
    }
}

// ------------------------------------------------------------- launchers ---
static int p3_cus()
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

bool conv3x3_supported(int dtype, int K, int N, int W)
{
    if (dtype != DT_BF16 || K > 128 || N > 128 || W > kP3MaxW || W < 1) return false;
    return p3_geom<bf16_t>(K, N, W).lds <= 160 * 1024;
}

int64_t conv3x3_partial_rows(int64_t m)
{
    const int64_t tiles = ceil_div(m, kP3BM);
    const int64_t g = p3_cus();
    return tiles < g ? tiles : g;
}

template <int NPC, int EK, bool BNG>
static hipError_t run_p3(const RowsParams &p, const P3Geom &g, hipStream_t s)
{
    // 32 output columns: eight waves of 16 rows; wider: 4 x 2 waves of 32 rows
    constexpr int WM = NPC == 32 ? 8 : 4;
    auto kern = k_conv3x3<bf16_t, NPC, WM, EK, BNG>;
    static bool attr_set = false;
    if (!attr_set) {
        const hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    const int grid = (int)conv3x3_partial_rows(p.m);
    const double e = 2.0, m = (double)p.m;
    double a = m * p.K;
    if (BNG) a *= 2.0;
    double out = m * p.N;
    if (EK == EK_STORE_ACC || EK == EK_RELUMASK || EK == EK_BNBWD) out += m * p.N;
    TraceScope tr(KC_CONV, KID_CONV_3X3, s, e * (a + out + 9.0 * p.K * p.N), 2.0 * m * 9.0 * p.K * p.N);
    hipLaunchKernelGGL(kern, dim3(grid), dim3(kP3Threads), g.lds, s, p, g);
    return hipGetLastError();
}

template <int EK, bool BNG>
static hipError_t run_p3_np(const RowsParams &p, const P3Geom &g, hipStream_t s)
{
    switch (g.NP) {
    case 32: return run_p3<32, EK, BNG>(p, g, s);
    case 64: return run_p3<64, EK, BNG>(p, g, s);
    default: return run_p3<128, EK, BNG>(p, g, s);
    }
}

template <bool BNG>
static hipError_t run_p3_ek(const RowsParams &p, const P3Geom &g, int ek, hipStream_t s)
{
    switch (ek) {
    case EK_STORE: return run_p3_np<EK_STORE, BNG>(p, g, s);
    case EK_STORE_ACC: return run_p3_np<EK_STORE_ACC, BNG>(p, g, s);
    case EK_STATS: return run_p3_np<EK_STATS, BNG>(p, g, s);
    case EK_RELUMASK: return run_p3_np<EK_RELUMASK, BNG>(p, g, s);
    default: return run_p3_np<EK_BNBWD, BNG>(p, g, s);
    }
}

hipError_t launch_conv3x3(const RowsParams &p, hipStream_t s)
{
    if (!p.a || !p.wraw || !p.y || p.taps != 9 || p.pro == PRO_POOLUP || !conv3x3_supported(p.dtype, p.K, p.N, p.w))
        return hipErrorInvalidValue;
    if (p.pro == PRO_BNRELU && (!p.p_mean || !p.p_gamma || !p.p_rstd || !p.p_beta)) return hipErrorInvalidValue;
    if (p.pro == PRO_BNGRAD && (!p.a2 || !p.p_mean || !p.p_rstd || !p.p_gamma || !p.p_dbeta || !p.p_dgamma))
        return hipErrorInvalidValue;
    if ((p.epi == EPI_STATS || p.epi == EPI_BNBWD) && !p.part) return hipErrorInvalidValue;
    if (p.epi == EPI_BNBWD && (!p.ex || !p.e_mean || !p.e_rstd || !p.e_gamma || !p.e_beta)) return hipErrorInvalidValue;
    if (p.epi == EPI_RELUMASK && !p.ex) return hipErrorInvalidValue;
    if ((int64_t)p.n * p.h * p.w != p.m || p.m < 1) return hipErrorInvalidValue;
    // 32-bit pixel indices and raw-buffer operand views: every span below 2^31 bytes
    const int64_t lim = (int64_t)1 << 31;
    if (p.m >= (lim >> 1) || (p.m * p.a_ldc + p.K) * 2 >= lim || (p.m * p.y_ldc + p.N) * 2 >= lim ||
        (p.a2 && (p.m * p.a2_ldc + p.K) * 2 >= lim) || (p.ex && (p.m * p.ex_ldc + p.N) * 2 >= lim))
        return hipErrorInvalidValue;
    const P3Geom g = p3_geom<bf16_t>(p.K, p.N, p.w);
    const int ek = epilogue_kind(p.epi, p.accumulate);
    if (p.pro == PRO_BNGRAD) return run_p3_ek<true>(p, g, ek, s);
    return run_p3_ek<false>(p, g, ek, s);
}

}  // namespace bnr
