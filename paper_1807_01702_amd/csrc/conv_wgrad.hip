// conv_wgrad.hip -- CONV weight gradient on the gfx950 matrix cores with the
// fission/fusion prologues on both operands.
//
//   dW[kh][kw][ci][co] = sum over pixels q of Z[q][ci] * G[q - off][co]
//
// Z is relu(bn(x)) recomputed from x on load (no stored activation), relu(x)
// or x itself; G is a dense gradient, the deferred BN input gradient
// k*(dy - a - xhat*b) formed from (dy, x) on load, or the 2x2 average-pooling
// gradient formed from the pooled gradient.  For 3x3 the tap shift is applied
// to G, so Z is read unshifted.
//
// GEMM view: M = 64 input channels x taps, N = output channels, K = pixels.
// K comes in chunks of 64 positions staged transposed in LDS (channel-major,
// pixel-contiguous) so that a lane's 8 consecutive k values are one 16-byte
// read.  3x3 chunks are R whole image rows in a zero-padded layout (one zero
// column on the left, zeros up to the padded width PW).  A workgroup owns one
// filter row kh, so the G operand of a chunk is the same R rows shifted by
// dh = kh - 1 (zero outside the image), laid out the same way: tap kw then
// reads G at offset 1 - kw from the Z position, out-of-image neighbours read
// the zeros, and only kw = 0 / 2 need a 2-byte realignment (four alignbyte
// ops on five dword reads).
// The next chunk's global loads are issued before the current chunk's matrix
// work.  S pixel splits write float32 partial tiles; a fixed-order sum gives
// dW (deterministic).
#include "common.hpp"
#include "kernels.hpp"
#include "mfma.hpp"
#include "tiles.hpp"
#include "trace.hpp"

namespace bnr {

template <typename T, int TAPS, int COT>
struct WgCfg {
    static constexpr int VEC = Elem<T>::VEC;
    static constexpr int PAD = 16 / (int)sizeof(T);
    static constexpr int ZSTR = kWgKC + PAD;
    static constexpr int GOFF = 8;                                    // zero guard in front of a G row
    static constexpr int GCOLS = kWgKC;                               // R * PW = 64
    static constexpr int GSTR = GOFF + GCOLS + 8 + PAD;
    static constexpr int ZITEMS = (kWgKC / 2) * (kWgCIT / VEC);       // pixel pairs x vectors
    static constexpr int GITEMS = (GCOLS / 2) * (COT / VEC);
    static constexpr int ZI = (ZITEMS + kThreads - 1) / kThreads;
    static constexpr int GI = (GITEMS + kThreads - 1) / kThreads;
};

// 8 consecutive storage elements starting at element s of an LDS row whose
// base is 16-byte aligned; s % 8 is the same for every lane of the call.
template <typename T> struct Shifted;
template <> struct Shifted<bf16_t> {
    __device__ static __forceinline__ bf16x8 load(const bf16_t *row, int s) {
        if ((s & 7) == 0) return Mfma<bf16_t>::load(row + s);
        uint32_t w[4];
        if ((s & 1) == 0) {
            const uint32_t *p = reinterpret_cast<const uint32_t *>(row + s);
            for (int i = 0; i < 4; i++) w[i] = p[i];
        } else {
            const uint32_t *p = reinterpret_cast<const uint32_t *>(row + s - 1);
            uint32_t v[5];
            for (int i = 0; i < 5; i++) v[i] = p[i];
            for (int i = 0; i < 4; i++) w[i] = __builtin_amdgcn_alignbyte(v[i + 1], v[i], 2);
        }
        return Mfma<bf16_t>::from_words(w);
    }
};
template <> struct Shifted<float> {
    __device__ static __forceinline__ float load(const float *row, int s) { return row[s]; }
};

// two pixels' values of one channel -> one LDS store
template <typename T> __device__ __forceinline__ void st_pair(T *dst, float a, float b);
template <> __device__ __forceinline__ void st_pair<bf16_t>(bf16_t *dst, float a, float b) {
    *reinterpret_cast<uint32_t *>(dst) = pack2bf(a, b);
}
template <> __device__ __forceinline__ void st_pair<float>(float *dst, float a, float b) {
    *reinterpret_cast<float2 *>(dst) = make_float2(a, b);
}

// K position of a chunk -> pixel index (or -1: a zero position)
struct ChunkGeo {
    int taps, H, W, R, PW;
    int64_t m, q0;     // 1x1: first pixel of the chunk
    int64_t img;       // 3x3: image of the chunk
    int h0;            // 3x3: first image row of the chunk
    __device__ int64_t zpix(int kp) const {
        if (taps == 1) {
            const int64_t q = q0 + kp;
            return q < m ? q : -1;
        }
        const int r = kp / PW, c = kp - r * PW;
        const int h = h0 + r;
        if (r >= R || h >= H || c < 1 || c > W) return -1;
        return (img * H + h) * W + (c - 1);
    }
    // G position (row r of the chunk, column c) -> pixel (h0 + r - dh, c - 1) or -1
    __device__ int64_t gpix(int gp, int dh) const {
        if (taps == 1) return zpix(gp);
        const int r = gp / PW, c = gp - r * PW;
        const int h = h0 + r - dh;
        if (r >= R || h < 0 || h >= H || c < 1 || c > W) return -1;
        return (img * H + h) * W + (c - 1);
    }
};

template <typename T, int TAPS, int COT, int WR, int WC>
__global__ __launch_bounds__(kThreads) void k_wgrad(WgradParams p, WgradPlan pl)
{
    using Cfg = WgCfg<T, TAPS, COT>;
    using M = Mfma<T>;
    constexpr int VEC = Cfg::VEC, ZSTR = Cfg::ZSTR, GSTR = Cfg::GSTR, GOFF = Cfg::GOFF;
    constexpr int RB = kWgCIT / 16 / WR;      // 16-row blocks of ci per wave
    constexpr int CB = COT / 16 / WC;         // 16-column blocks of co per wave
    static_assert(WR * WC == 4, "four waves");
    __shared__ __align__(16) T Zt[kWgCIT * ZSTR];
    __shared__ __align__(16) T Gt[COT * GSTR];
    __shared__ float zc[3][kWgCIT];           // c0, c1, centre (float32 data: x - K below)
    __shared__ float gc[4][COT];              // A, B, C, centre of gx

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wr = wave / WC, wc = wave % WC;
    const int n_out = pl.ci_tiles * pl.kh_tiles * pl.co_tiles;
    const int lid = xcd_remap(blockIdx.x, gridDim.x);
    const int ot = lid % n_out, split = lid / n_out;
    const int co_t = ot % pl.co_tiles, kh_t = (ot / pl.co_tiles) % pl.kh_tiles, ci_t = ot / (pl.co_tiles * pl.kh_tiles);
    const int ci0 = ci_t * kWgCIT, co0 = co_t * COT;
    const int C_in = p.c_in, C_out = p.c_out;
    const int64_t m = p.m;
    const int gcols = kWgKC;
    const int dh = TAPS == 3 ? kh_t - 1 : 0;

    if (tid < kWgCIT) {
        const int c = ci0 + tid;
        if (p.a_mode == 1 && c < C_in) {        // the forward's y = x c0 + c1
            bn_coef(p.a_gamma[c], p.a_beta[c], p.a_mean[c], p.a_rstd[c], zc[0][tid], zc[1][tid]);
            zc[2][tid] = bn_centre<T>(p.a_ctr, c);
        }
    }
    if (tid < COT) {
        const int c = co0 + tid;
        if (p.gsrc == GB_BNGRAD && c < C_out) {
            deferred_coef(p.g_split, c, 1.0f / (float)m, p.g_gamma, p.g_mean, p.g_rstd, p.g_dgamma, p.g_dbeta,
                          p.g_alpha, p.g_betap, gc[0][tid], gc[1][tid], gc[2][tid]);
            gc[3][tid] = bn_centre<T>(p.g_ctr, c);
        }
    }
    // zero the G guards and the columns beyond gcols once; staging never writes them
    for (int i = tid; i < COT * GSTR; i += kThreads) {
        const int col = i % GSTR;
        if (col < GOFF || col >= GOFF + gcols) Gt[i] = T(0);
    }

    f32x4 acc[TAPS][RB][CB];
    for (int t = 0; t < TAPS; t++)
        for (int rb = 0; rb < RB; rb++)
            for (int cb = 0; cb < CB; cb++) acc[t][rb][cb] = f32x4{0.f, 0.f, 0.f, 0.f};

    const T *xs = reinterpret_cast<const T *>(p.x);
    const T *gs = reinterpret_cast<const T *>(p.g);
    const T *gxs = reinterpret_cast<const T *>(p.gx);
    const int64_t ch_begin = (int64_t)split * pl.chunks_per_split;
    const int64_t ch_end = min(pl.nchunks, ch_begin + pl.chunks_per_split);
    const int zitems = Cfg::ZITEMS;
    const int gitems = (gcols / 2) * (COT / VEC);

    // ---- register stage of one chunk (raw loads; transforms at LDS store) ----
    vec16 zr[Cfg::ZI][2], gr[Cfg::GI][2], gx[Cfg::GI][2];
    auto geo_of = [&](int64_t ch) {
        ChunkGeo g;
        g.taps = TAPS; g.H = p.h; g.W = p.w; g.R = pl.R; g.PW = pl.PW; g.m = m;
        if (TAPS == 1) { g.q0 = ch * kWgKC; g.img = 0; g.h0 = 0; }
        else {
            g.q0 = 0;
            g.img = ch / pl.chunks_per_image;
            g.h0 = (int)(ch - g.img * pl.chunks_per_image) * pl.R;
        }
        return g;
    };
    auto load_chunk = [&](int64_t ch) {
        const ChunkGeo g = geo_of(ch);
        for (int j = 0; j < Cfg::ZI; j++) {
            const int i = tid + j * kThreads;
            const int v = i % (kWgCIT / VEC), pr = i / (kWgCIT / VEC);
            const int c = ci0 + v * VEC;
            for (int h2 = 0; h2 < 2; h2++) {
                const int64_t q = i < zitems ? g.zpix(2 * pr + h2) : -1;
                zr[j][h2] = (q >= 0 && c < C_in) ? ldg16(xs + q * p.x_ldc + c) : zero16();
            }
        }
        for (int j = 0; j < Cfg::GI; j++) {
            const int i = tid + j * kThreads;
            const int v = i % (COT / VEC), pr = i / (COT / VEC);
            const int c = co0 + v * VEC;
            for (int h2 = 0; h2 < 2; h2++) {
                const int64_t q = i < gitems ? g.gpix(2 * pr + h2, dh) : -1;
                vec16 a = zero16(), b = zero16();
                if (q >= 0 && c < C_out) {
                    if (p.gsrc == GB_DENSE) {
                        a = ldg16(gs + q * p.g_ldc + c);
                    } else if (p.gsrc == GB_BNGRAD) {
                        a = ldg16(gs + q * p.g_ldc + c);
                        b = ldg16(gxs + q * p.gx_ldc + c);
                    } else {
                        const int64_t img = q / ((int64_t)p.h * p.w);
                        const int rem = (int)(q - img * p.h * p.w);
                        const int y = rem / p.w, xx = rem - y * p.w;
                        const int64_t qq = (img * (p.h / 2) + y / 2) * (p.w / 2) + xx / 2;
                        a = ldg16(gs + qq * p.g_ldc + c);
                    }
                }
                gr[j][h2] = a;
                gx[j][h2] = b;
            }
        }
    };
    auto store_chunk = [&](int64_t ch) {
        const ChunkGeo g = geo_of(ch);
        for (int j = 0; j < Cfg::ZI; j++) {
            const int i = tid + j * kThreads;
            if (i >= zitems) break;
            const int v = i % (kWgCIT / VEC), pr = i / (kWgCIT / VEC);
            const int cl = v * VEC;
            float f[2][VEC];
            for (int h2 = 0; h2 < 2; h2++) {
                Elem<T>::unpack(zr[j][h2], f[h2]);
                const bool valid = g.zpix(2 * pr + h2) >= 0 && ci0 + cl < C_in;
                if (p.a_mode == 1)
                    for (int e = 0; e < VEC; e++) {
                        const float t = bn_lin(f[h2][e] - zc[2][cl + e], zc[0][cl + e], zc[1][cl + e]);
                        f[h2][e] = valid && t > 0.f ? t : 0.f;
                    }
                else if (p.a_mode == 2)
                    for (int e = 0; e < VEC; e++) f[h2][e] = f[h2][e] > 0.f ? f[h2][e] : 0.f;
            }
            for (int e = 0; e < VEC; e++) st_pair<T>(Zt + (cl + e) * ZSTR + 2 * pr, f[0][e], f[1][e]);
        }
        for (int j = 0; j < Cfg::GI; j++) {
            const int i = tid + j * kThreads;
            if (i >= gitems) break;
            const int v = i % (COT / VEC), pr = i / (COT / VEC);
            const int cl = v * VEC;
            float f[2][VEC];
            for (int h2 = 0; h2 < 2; h2++) {
                Elem<T>::unpack(gr[j][h2], f[h2]);
                if (p.gsrc == GB_BNGRAD) {
                    const bool valid = g.gpix(2 * pr + h2, dh) >= 0 && co0 + cl < C_out;
                    float x[VEC];
                    Elem<T>::unpack(gx[j][h2], x);
                    for (int e = 0; e < VEC; e++) {
                        const float d = __builtin_fmaf(gc[0][cl + e], f[h2][e],
                                                       __builtin_fmaf(gc[1][cl + e], x[e] - gc[3][cl + e], gc[2][cl + e]));
                        f[h2][e] = valid ? d : 0.f;
                    }
                } else if (p.gsrc == GB_POOLUP) {
                    for (int e = 0; e < VEC; e++) f[h2][e] *= 0.25f;
                }
            }
            for (int e = 0; e < VEC; e++) st_pair<T>(Gt + (cl + e) * GSTR + GOFF + 2 * pr, f[0][e], f[1][e]);
        }
    };

    if (ch_begin < ch_end) load_chunk(ch_begin);
    __syncthreads();
    for (int64_t ch = ch_begin; ch < ch_end; ch++) {
        store_chunk(ch);
        __syncthreads();
        if (ch + 1 < ch_end) load_chunk(ch + 1);
        // ---- matrix cores ----
        for (int ks = 0; ks < kWgKC / M::KSTEP; ks++) {
            const int kq = ks * M::KSTEP + (lane >> 4) * M::KPL;
            typename M::frag a[RB];
            for (int rb = 0; rb < RB; rb++) a[rb] = M::load(Zt + ((wr * RB + rb) * 16 + (lane & 15)) * ZSTR + kq);
            for (int t = 0; t < TAPS; t++) {
                // G position of Z position kq for tap (kh_t, kw = t): 1 - kw
                const int off = TAPS == 3 ? 1 - t : 0;
                for (int cb = 0; cb < CB; cb++) {
                    const T *row = Gt + ((wc * CB + cb) * 16 + (lane & 15)) * GSTR;
                    const typename M::frag b = Shifted<T>::load(row, GOFF + off + kq);
                    for (int rb = 0; rb < RB; rb++) M::mma(acc[t][rb][cb], a[rb], b);
                }
            }
        }
        __syncthreads();
    }

    // ---- partial tile (or dW directly when there is one split) ----
    float *dst = pl.splits == 1 ? p.dw : p.part + (int64_t)split * p.k * p.k * C_in * C_out;
    for (int t = 0; t < TAPS; t++) {
        const int tap = TAPS == 3 ? kh_t * 3 + t : 0;
        for (int rb = 0; rb < RB; rb++)
            for (int cb = 0; cb < CB; cb++)
                for (int i = 0; i < 4; i++) {
                    const int ci = ci0 + (wr * RB + rb) * 16 + (lane >> 4) * 4 + i;
                    const int co = co0 + (wc * CB + cb) * 16 + (lane & 15);
                    if (ci < C_in && co < C_out) dst[((int64_t)tap * C_in + ci) * C_out + co] = acc[t][rb][cb][i];
                }
    }
}

// ---------------------------------------------------------------------------
// bf16 weight gradient with transposing LDS reads (gfx950 ds_read_b64_tr_b16).
// Z and G are staged row-major exactly as they arrive from HBM (one row per K
// position, 16-byte channel vectors), after the prologue transform; a
// matrix-core fragment (8 consecutive K positions of one channel per lane) is
// two transposing 8-byte reads.  Within a group of 16 lanes, lane j reads the
// 4 channels 4 (j % 4) .. +3 of row j / 4 and lane i receives channel i of
// rows 0..3 (layout checked on the device).  For 3x3 every tap is a row
// offset into the staged Z, so all nine taps share the G fragments.

// Two workgroups per CU wherever the operand registers allow it without
// spilling (all but the 64-channel 3x3 tiles, whose nine accumulator sets
// need one workgroup's whole register file).
template <int TAPS, int CIT, int COT, int WCI, int GS>
__global__ __launch_bounds__(kThreads, (TAPS == 3 && COT == 64) ? 1 : 2) void k_wgrad_tr(WgradParams p, WgTrPlan pl)
{
    using T = bf16_t;
    using M = Mfma<T>;
    constexpr int VEC = 8;
    constexpr int WCO = 4 / WCI;
    constexpr int RB = CIT / 16 / WCI, CB = COT / 16 / WCO;
    constexpr int ZP = CIT + 8, GP = COT + 8;                     // LDS row pitches (elements)
    constexpr int VZ = CIT / VEC, VG = COT / VEC;                 // vectors per staged row
    constexpr int KQMAX = TAPS == 3 ? 128 : kWgTrKQ1;            // positions per chunk (upper bound)
    constexpr int ZRMAX = TAPS == 3 ? KQMAX + 2 * (kWgMaxW3 + 2) + 2 : KQMAX;
    constexpr int NZ = (ZRMAX * VZ + kThreads - 1) / kThreads;
    constexpr int NG = (KQMAX * VG + kThreads - 1) / kThreads;
    constexpr int NGX = GS == GB_BNGRAD ? NG : 1;
    static_assert(WCI * WCO == 4 && RB >= 1 && CB >= 1, "wave layout");
    extern __shared__ __align__(16) unsigned char smem[];
    T *Zs = reinterpret_cast<T *>(smem);                          // [zrows][ZP]
    T *Gs = Zs + (size_t)(pl.zrows + 1) * ZP;                     // [KQ + 1][GP]
    float *gco = reinterpret_cast<float *>(Gs + (size_t)(pl.KQ + 1) * GP);   // BNGRAD coefficients [3][COT]

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wci = wave % WCI, wco = wave / WCI;
    const int n_out = pl.ci_tiles * pl.co_tiles;
    const int lid = xcd_remap(blockIdx.x, gridDim.x);
    const int ot = lid % n_out, split = lid / n_out;
    const int co_t = ot % pl.co_tiles, ci_t = ot / pl.co_tiles;
    const int ci0 = ci_t * CIT, co0 = co_t * COT;
    const int C_in = p.c_in, C_out = p.c_out, H = p.h, W = p.w;
    const int64_t m = p.m;
    const int PW = pl.PW, KQ = pl.KQ, ZR = pl.zrows;

    // per-thread channel vectors (fixed: 256 is a multiple of VZ and VG)
    const int vz = tid % VZ, vg = tid % VG;
    const int cz = ci0 + vz * VEC, cg = co0 + vg * VEC;
    const bool zc_ok = cz < C_in, gc_ok = cg < C_out;
    // (the deferred-gradient parameters first, then one branch around all 32
    // operand parameters, so every load is in flight together: a branch per
    // channel made eight round trips)
    float gq0 = 0.f, gq1 = 0.f, gq2 = 0.f, gq3 = 0.f, gq4 = 0.f;
    const bool gco_ld = GS == GB_BNGRAD && tid < COT && co0 + tid < C_out;
    if (gco_ld) {
        const int c = co0 + tid;
        gq1 = p.g_mean[c]; gq2 = p.g_rstd[c];
        if (p.g_split) { gq0 = p.g_alpha[c]; gq3 = p.g_betap[c]; }
        else { gq0 = p.g_gamma[c]; gq3 = p.g_dgamma[c]; gq4 = p.g_dbeta[c]; }
    }
    float za[VEC], zb[VEC];
    #pragma unroll
    for (int e = 0; e < VEC; e++) { za[e] = 1.f; zb[e] = 0.f; }
    if (p.a_mode == 1 && zc_ok) {
        float ga[VEC], be[VEC], mu[VEC], rs[VEC];
        #pragma unroll
        for (int e = 0; e < VEC; e++) {
            ga[e] = p.a_gamma[cz + e]; be[e] = p.a_beta[cz + e]; mu[e] = p.a_mean[cz + e]; rs[e] = p.a_rstd[cz + e];
        }
        #pragma unroll
        for (int e = 0; e < VEC; e++) bn_coef(ga[e], be[e], mu[e], rs[e], za[e], zb[e]);
    }
    // deferred-gradient coefficients in LDS (registers are the occupancy limit of the 3x3 variants)
    if (GS == GB_BNGRAD && tid < COT) {
        float A = 0.f, Bc = 0.f, Cc = 0.f;
        if (gco_ld) deferred_coef_of(p.g_split, 1.0f / (float)m, gq0, gq1, gq2, gq3, gq4, A, Bc, Cc);
        gco[tid] = A; gco[COT + tid] = Bc; gco[2 * COT + tid] = Cc;
    }
    __syncthreads();

    // raw-buffer views (launcher: every span below 2^31 bytes)
    const __amdgpu_buffer_rsrc_t xbuf = buf_view(p.x, (uint32_t)(((m - 1) * p.x_ldc + C_in) * 2));
    const int64_t gpix = GS == GB_POOLUP ? m / 4 : m;
    const __amdgpu_buffer_rsrc_t gbuf = buf_view(p.g, (uint32_t)(((gpix - 1) * p.g_ldc + C_out) * 2));
    const __amdgpu_buffer_rsrc_t gxbuf = buf_view(GS == GB_BNGRAD ? p.gx : p.g,
                                                  GS == GB_BNGRAD ? (uint32_t)(((m - 1) * p.gx_ldc + C_out) * 2) : 0u);

    // The staged rows of this thread are the same in every chunk, so the
    // 3x3 row -> pixel map is split once into a row offset r (image rows
    // below the chunk's first row; a large negative value for a row that is
    // never a pixel) and a pixel offset r W + col - 1; per chunk a pixel is
    // then one add and one range test (no division in the loop).
    constexpr int kNever = -(1 << 28);
    int zrr[NZ], zro[NZ], grr[NG], gro[NG];
    #pragma unroll
    for (int j = 0; j < NZ; j++) {
        zrr[j] = kNever; zro[j] = 0;
        if (TAPS == 3) {
            const int row = tid / VZ + j * (kThreads / VZ);
            const int q = row - (PW + 1);
            const int r = (q + 2 * PW) / PW - 2;                  // floor(q / PW) for q >= -2 PW
            const int col = q - r * PW;
            zrr[j] = row < ZR && col >= 1 && col <= W ? r : kNever;
            zro[j] = r * W + col - 1;
        }
    }
    #pragma unroll
    for (int j = 0; j < NG; j++) {
        grr[j] = kNever; gro[j] = 0;
        if (TAPS == 3) {
            const int row = tid / VG + j * (kThreads / VG);
            const int r = row / PW, col = row - r * PW;
            grr[j] = row < KQ && r < pl.R && col >= 1 && col <= W ? r : kNever;
            gro[j] = r * W + col - 1;
        }
    }
    // pixel of staged row j (Z side: zside) of a chunk whose first pixel is
    // base (3x3: (img H + h0) W; 1x1: img 64), or -1; 32-bit (launcher: every
    // pixel index below 2^30), selects only
    auto pix = [&](int base, int h0, int j, bool zside) __attribute__((always_inline)) -> int {
        if (TAPS == 1) {
            const int q = tid / (zside ? VZ : VG) + j * (kThreads / (zside ? VZ : VG));
            const int pp = base + q;
            return ((q < KQ) & (pp < (int)m)) ? pp : -1;
        }
        const int r = zside ? zrr[j] : grr[j];
        const int o = zside ? zro[j] : gro[j];
        return (unsigned)(h0 + r) < (unsigned)H ? base + o : -1;
    };
    // 32-bit element offsets (launcher: every operand span below 2^31 bytes)
    const int xl = (int)p.x_ldc, gl = (int)p.g_ldc, gxl = (int)p.gx_ldc;
    auto chunk_pix0 = [&](int64_t img, int h0) __attribute__((always_inline)) -> int {
        return TAPS == 3 ? (int)((img * H + h0) * W) : (int)(img * KQMAX);
    };

    vec16 zr[NZ], gr[NG], gx[NGX];
    auto load_chunk = [&](int64_t img, int h0) __attribute__((always_inline)) {
        const int base = chunk_pix0(img, h0);
        #pragma unroll
        for (int j = 0; j < NZ; j++) {
            const int row = tid / VZ + j * (kThreads / VZ);
            const int q = pix(base, h0, j, true);
            const bool ok = (row < ZR) & (q >= 0) & zc_ok;
            zr[j] = bld16(xbuf, ok ? (uint32_t)(q * xl + cz) * 2u : kBufOff);
        }
        #pragma unroll
        for (int j = 0; j < NG; j++) {
            const int row = tid / VG + j * (kThreads / VG);
            const int q = pix(base, h0, j, false);
            const bool ok = (row < KQ) & (q >= 0) & gc_ok;
            if (GS == GB_POOLUP) {
                // 32-bit quotients (launcher: every pixel index below 2^31)
                const int qi = q > 0 ? (int)q : 0;
                const int im = qi / (H * W);
                const int rem = qi - im * H * W;
                const int y = rem / W, xx = rem - y * W;
                const int64_t qq = ((int64_t)im * (H / 2) + y / 2) * (W / 2) + xx / 2;
                gr[j] = bld16(gbuf, ok ? (uint32_t)((int)qq * gl + cg) * 2u : kBufOff);
            } else {
                gr[j] = bld16(gbuf, ok ? (uint32_t)(q * gl + cg) * 2u : kBufOff);
            }
            if (GS == GB_BNGRAD) gx[j < NGX ? j : 0] = bld16(gxbuf, ok ? (uint32_t)(q * gxl + cg) * 2u : kBufOff);
        }
    };
    // Prologue transforms as straight-line code: the ReLU is max(t, zlo)
    // (zlo = -inf without one), invalid rows are zeroed on the packed words,
    // and rows past the staged range go to a junk row (no per-row branch).
    const float zlo = p.a_mode != 0 ? 0.f : -__builtin_inff();
    auto store_chunk = [&](int64_t img, int h0) __attribute__((always_inline)) {
        const int base = chunk_pix0(img, h0);
        #pragma unroll
        for (int j = 0; j < NZ; j++) {
            const int row = tid / VZ + j * (kThreads / VZ);
            const bool valid = (row < ZR) & (pix(base, h0, j, true) >= 0) & zc_ok;
            float f[VEC];
            Elem<T>::unpack(zr[j], f);
            #pragma unroll
            for (int e = 0; e < VEC; e++) f[e] = __builtin_fmaxf(bn_lin(f[e], za[e], zb[e]), zlo);
            vec16 out = Elem<T>::pack(f);
            #pragma unroll
            for (int i = 0; i < 4; i++) out.u[i] = valid ? out.u[i] : 0u;
            *reinterpret_cast<vec16 *>(Zs + (row < ZR ? row : ZR) * ZP + vz * VEC) = out;
        }
        // (this thread's G channel vector is the same in every slot: its
        // deferred-gradient coefficients are read once per chunk)
        float gA[VEC], gB[VEC], gC[VEC];
        if (GS == GB_BNGRAD) {
            lds_f8(gco + vg * VEC, gA);
            lds_f8(gco + COT + vg * VEC, gB);
            lds_f8(gco + 2 * COT + vg * VEC, gC);
        }
        #pragma unroll
        for (int j = 0; j < NG; j++) {
            const int row = tid / VG + j * (kThreads / VG);
            vec16 out = gr[j];
            if (GS == GB_BNGRAD) {
                const bool valid = (row < KQ) & (pix(base, h0, j, false) >= 0) & gc_ok;
                float d[VEC], x[VEC];
                Elem<T>::unpack(gr[j], d);
                Elem<T>::unpack(gx[j < NGX ? j : 0], x);
                #pragma unroll
                for (int e = 0; e < VEC; e++) d[e] = __builtin_fmaf(gA[e], d[e], __builtin_fmaf(gB[e], x[e], gC[e]));
                out = Elem<T>::pack(d);
                #pragma unroll
                for (int i = 0; i < 4; i++) out.u[i] = valid ? out.u[i] : 0u;
            } else if (GS == GB_POOLUP) {
                float d[VEC];
                Elem<T>::unpack(gr[j], d);
                #pragma unroll
                for (int e = 0; e < VEC; e++) d[e] *= 0.25f;
                out = Elem<T>::pack(d);
            }
            *reinterpret_cast<vec16 *>(Gs + (row < KQ ? row : KQ) * GP + vg * VEC) = out;
        }
    };

    f32x4 acc[TAPS * TAPS][RB][CB];
    #pragma unroll
    for (int t = 0; t < TAPS * TAPS; t++)
        #pragma unroll
        for (int rb = 0; rb < RB; rb++)
            #pragma unroll
            for (int cb = 0; cb < CB; cb++) acc[t][rb][cb] = f32x4{0.f, 0.f, 0.f, 0.f};

    // this lane's transposing-read offsets (elements)
    const int g16 = lane >> 4, j16 = lane & 15;
    const T *za_base = Zs + (8 * g16 + (j16 >> 2)) * ZP + 4 * (j16 & 3) + wci * RB * 16;
    const T *gb_base = Gs + (8 * g16 + (j16 >> 2)) * GP + 4 * (j16 & 3) + wco * CB * 16;

    // chunk positions (image, first row) advanced incrementally
    const int64_t ch_begin = (int64_t)split * pl.chunks_per_split;
    const int64_t ch_end = min(pl.nchunks, ch_begin + pl.chunks_per_split);
    struct Pos { int64_t img; int h0, cin; };
    auto first = [&]() -> Pos {
        Pos q;
        if (TAPS == 3) {
            q.img = ch_begin / pl.chunks_per_image;
            q.cin = (int)(ch_begin - q.img * pl.chunks_per_image);
            q.h0 = q.cin * pl.R;
        } else {
            q.img = ch_begin; q.cin = 0; q.h0 = 0;
        }
        return q;
    };
    auto advance = [&](Pos &q) __attribute__((always_inline)) {
        if (TAPS == 3) {
            q.cin++; q.h0 += pl.R;
            if (q.cin == pl.chunks_per_image) { q.cin = 0; q.h0 = 0; q.img++; }
        } else {
            q.img++;
        }
    };
    Pos ps = first(), pn = ps;
    if (ch_begin < ch_end) load_chunk(pn.img, pn.h0);
    for (int64_t ch = ch_begin; ch < ch_end; ch++) {
        store_chunk(ps.img, ps.h0);
        __syncthreads();
        advance(pn);
        if (ch + 1 < ch_end) load_chunk(pn.img, pn.h0);
        advance(ps);
        for (int kq = 0; kq < KQ; kq += M::KSTEP) {
            typename M::frag b[CB];
            #pragma unroll
            for (int cb = 0; cb < CB; cb++) b[cb] = tr_frag(gb_base + kq * GP + cb * 16, GP);
            #pragma unroll
            for (int t = 0; t < TAPS * TAPS; t++) {
                const int toff = TAPS == 3 ? (t / 3) * PW + (t % 3) : 0;
                #pragma unroll
                for (int rb = 0; rb < RB; rb++) {
                    const typename M::frag a = tr_frag(za_base + (kq + toff) * ZP + rb * 16, ZP);
                    #pragma unroll
                    for (int cb = 0; cb < CB; cb++) M::mma(acc[t][rb][cb], a, b[cb]);
                }
            }
        }
        __syncthreads();
    }

    // ---- partial tile (or dW directly when there is one split) ----
    float *dst = pl.splits == 1 ? p.dw : p.part + (int64_t)split * p.k * p.k * C_in * C_out;
    #pragma unroll
    for (int t = 0; t < TAPS * TAPS; t++)
        #pragma unroll
        for (int rb = 0; rb < RB; rb++)
            #pragma unroll
            for (int cb = 0; cb < CB; cb++)
                #pragma unroll
                for (int i = 0; i < 4; i++) {
                    const int ci = ci0 + (wci * RB + rb) * 16 + (lane >> 4) * 4 + i;
                    const int co = co0 + (wco * CB + cb) * 16 + (lane & 15);
                    if (ci < C_in && co < C_out) dst[((int64_t)t * C_in + ci) * C_out + co] = acc[t][rb][cb][i];
                }
}

// ------------------------------------------------------------- launchers ---
static bool wgrad_tr_ok(int dtype, int64_t m, int h, int w, int64_t x_ldc, int64_t g_ldc, int64_t gx_ldc, int k)
{
    if (dtype != DT_BF16 || (k == 3 && w > kWgMaxW3)) return false;
    const int64_t lim = (int64_t)1 << 31;
    return (m * x_ldc) * 2 < lim && (m * g_ldc) * 2 < lim && (m * gx_ldc) * 2 < lim && h >= 1 && w >= 1;
}

size_t wgrad_ws_bytes(int dtype, int64_t m, int n, int h, int w, int c_in, int c_out, int k)
{
    const WgradPlan pl = wgrad_plan(m, n, h, w, c_in, c_out, k, dtype == DT_BF16 ? 2 : 4);
    const WgTrPlan tp = wgrad_tr_plan(m, n, h, w, c_in, c_out, k);
    const int64_t s = dtype == DT_BF16 ? (pl.splits > tp.splits ? pl.splits : tp.splits) : pl.splits;
    if (s <= 1) return 0;
    return (size_t)s * k * k * c_in * c_out * sizeof(float);
}

template <int TAPS, int CIT, int COT, int WCI>
static hipError_t run_wgrad_tr(const WgradParams &p, const WgTrPlan &pl, hipStream_t s)
{
    const int64_t blocks = (int64_t)pl.ci_tiles * pl.co_tiles * pl.splits;
    const size_t lds = ((size_t)(pl.zrows + 1) * (CIT + 8) + (size_t)(pl.KQ + 1) * (COT + 8)) * 2 + 3 * COT * sizeof(float);
    const double m = (double)p.m;
    double g = m * p.c_out;
    if (p.gsrc == GB_BNGRAD) g *= 2.0;
    if (p.gsrc == GB_POOLUP) g /= 4.0;
    const double dwb = (double)p.k * p.k * p.c_in * p.c_out;
    TraceScope tr(KC_WGRAD, TAPS == 3 ? KID_WGRAD_3X3 : KID_WGRAD_1X1, s, 2.0 * (m * p.c_in + g) + 4.0 * dwb,
                  2.0 * m * dwb);
    if (p.gsrc == GB_BNGRAD)
        hipLaunchKernelGGL((k_wgrad_tr<TAPS, CIT, COT, WCI, GB_BNGRAD>), dim3((unsigned)blocks), dim3(kThreads), lds, s, p, pl);
    else if (p.gsrc == GB_POOLUP)
        hipLaunchKernelGGL((k_wgrad_tr<TAPS, CIT, COT, WCI, GB_POOLUP>), dim3((unsigned)blocks), dim3(kThreads), lds, s, p, pl);
    else
        hipLaunchKernelGGL((k_wgrad_tr<TAPS, CIT, COT, WCI, GB_DENSE>), dim3((unsigned)blocks), dim3(kThreads), lds, s, p, pl);
    return hipGetLastError();
}

static hipError_t dispatch_wgrad_tr(const WgradParams &p, const WgTrPlan &pl, hipStream_t s)
{
    if (pl.k == 3) return pl.cot == 32 ? run_wgrad_tr<3, 64, 32, 4>(p, pl, s) : run_wgrad_tr<3, 64, 64, 4>(p, pl, s);
    if (pl.cit == 64) {
        if (pl.cot == 32) return run_wgrad_tr<1, 64, 32, 2>(p, pl, s);
        if (pl.cot == 64) return run_wgrad_tr<1, 64, 64, 2>(p, pl, s);
        return run_wgrad_tr<1, 64, 128, 1>(p, pl, s);
    }
    if (pl.cot == 32) return run_wgrad_tr<1, 128, 32, 4>(p, pl, s);
    if (pl.cot == 64) return run_wgrad_tr<1, 128, 64, 2>(p, pl, s);
    return run_wgrad_tr<1, 128, 128, 2>(p, pl, s);
}

template <typename T, int TAPS, int COT, int WR, int WC>
static hipError_t run_wgrad(const WgradParams &p, const WgradPlan &pl, hipStream_t s)
{
    const int64_t blocks = (int64_t)pl.ci_tiles * pl.kh_tiles * pl.co_tiles * pl.splits;
    const double e = sizeof(T), m = (double)p.m;
    double g = m * p.c_out;                                       // gradient operand
    if (p.gsrc == GB_BNGRAD) g *= 2.0;                            // dy and x
    if (p.gsrc == GB_POOLUP) g /= 4.0;                            // pooled gradient
    const double dwb = (double)p.k * p.k * p.c_in * p.c_out;
    TraceScope tr(KC_WGRAD, TAPS == 3 ? KID_WGRAD_3X3 : KID_WGRAD_1X1, s, e * (m * p.c_in + g) + 4.0 * dwb,
                  2.0 * m * dwb);
    hipLaunchKernelGGL((k_wgrad<T, TAPS, COT, WR, WC>), dim3((unsigned)blocks), dim3(kThreads), 0, s, p, pl);
    return hipGetLastError();
}

template <typename T>
static hipError_t dispatch_wgrad(const WgradParams &p, const WgradPlan &pl, hipStream_t s)
{
    if (p.k == 3) return pl.cot == 32 ? run_wgrad<T, 3, 32, 4, 1>(p, pl, s) : run_wgrad<T, 3, 64, 4, 1>(p, pl, s);
    if (pl.cot == 32) return run_wgrad<T, 1, 32, 4, 1>(p, pl, s);
    if (pl.cot == 64) return run_wgrad<T, 1, 64, 2, 2>(p, pl, s);
    return run_wgrad<T, 1, 128, 1, 4>(p, pl, s);
}

hipError_t launch_wgrad(const WgradParams &p, hipStream_t s, int64_t *splits_out)
{
    if (!p.x || !p.g || !p.dw) return hipErrorInvalidValue;
    if (p.a_mode == 1 && (!p.a_mean || !p.a_gamma || !p.a_rstd || !p.a_beta)) return hipErrorInvalidValue;
    if (p.gsrc == GB_BNGRAD && (!p.gx || !p.g_mean || !p.g_rstd ||
                                (p.g_split ? (!p.g_alpha || !p.g_betap) : (!p.g_gamma || !p.g_dbeta || !p.g_dgamma))))
        return hipErrorInvalidValue;
    if (p.k == 3 && p.w > kWgMaxW3) return hipErrorInvalidValue;
    if (wgrad_tr_ok(p.dtype, p.m, p.h, p.w, p.x_ldc, p.g_ldc, p.gsrc == GB_BNGRAD ? p.gx_ldc : 0, p.k)) {
        const WgTrPlan tp = wgrad_tr_plan(p.m, p.n, p.h, p.w, p.c_in, p.c_out, p.k);
        if (tp.splits > 1 && (!p.part || !p.red)) return hipErrorInvalidValue;
        const hipError_t e = dispatch_wgrad_tr(p, tp, s);
        if (splits_out) *splits_out = tp.splits;
        if (e != hipSuccess || tp.splits <= 1 || splits_out) return e;
        return launch_sum_partials(p.part, tp.splits, (int64_t)p.k * p.k * p.c_in * p.c_out, p.dw, p.red, s);
    }
    const WgradPlan pl = wgrad_plan(p.m, p.n, p.h, p.w, p.c_in, p.c_out, p.k, p.dtype == DT_BF16 ? 2 : 4);
    if (pl.splits > 1 && (!p.part || !p.red)) return hipErrorInvalidValue;
    const hipError_t e = p.dtype == DT_BF16 ? dispatch_wgrad<bf16_t>(p, pl, s) : dispatch_wgrad<float>(p, pl, s);
    if (splits_out) *splits_out = pl.splits;
    if (e != hipSuccess || pl.splits <= 1 || splits_out) return e;
    return launch_sum_partials(p.part, pl.splits, (int64_t)p.k * p.k * p.c_in * p.c_out, p.dw, p.red, s);
}

}  // namespace bnr
