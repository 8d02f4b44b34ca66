// net_ends.hip -- the layers at the two ends of a DenseNet training step.
//
//  * First CONV (7x7, stride 2, pad 3) with the sub-BN1 statistics epilogue
//    of the BN after it, and its weight gradient with the BN input gradient
//    formed on load (Sec. 3.2 fission/fusion applied to the network's first
//    layer; Sec. 3.1 names the 7x7 first CONV of DenseNet-121).
//  * BN -> ReLU -> 3x3/2 max pooling: forward with sub-BN2 + ReLU applied
//    while the pooling reads its input and the statistics of the pooled
//    output (the block input) in the same pass; backward with the ReLU mask
//    and the BN reductions in the pooling-gradient pass.
//  * Classifier head: BN -> ReLU -> global average pooling -> FC -> softmax
//    cross-entropy, forward and backward.
//
// First CONV on the matrix cores (bf16).  The image is staged in LDS with
// four channels per pixel (8 bytes; channels >= c_in read as 0), so for a
// filter row kh the 7 taps x 4 channels of one output pixel are 28
// consecutive elements at pixel 2*ow of the staged input row: a K step of 32
// is one filter row (tap slot 7 has zero weights) and a 16x16x32 fragment is
// one 16-byte LDS read per lane.  The weight fragments of all 7 filter rows
// stay in registers for the whole persistent loop.
#include "common.hpp"
#include "kernels.hpp"
#include "mfma.hpp"
#include "tiles.hpp"
#include "trace.hpp"

namespace bnr {

namespace {

constexpr int kSK = kStemK;                  // 7 taps per filter row
constexpr int kSIR = 2 * kStemRows + kSK - 2;     // staged input rows per item (9)
constexpr int kSPitch = 72;                  // LDS pitch (elements) of 64-channel rows
constexpr int kSKB = 2 * kSK;                // 16-wide k blocks of the weight gradient (14)

__host__ __device__ __forceinline__ int stem_rpx(int wo) { return 2 * wo + 6; }

// Item = (image, kStemRows consecutive output rows).
struct StemItem { int n, oh0, rows, pv; };
__device__ __forceinline__ StemItem stem_item(const StemParams &p, int64_t it)
{
    const int per = (p.ho + kStemRows - 1) / kStemRows;
    StemItem s;
    s.n = (int)(it / per);
    s.oh0 = (int)(it - (int64_t)s.n * per) * kStemRows;
    s.rows = min(kStemRows, p.ho - s.oh0);
    s.pv = s.rows * p.wo;
    return s;
}

// Stage the input rows of an item: row r <-> image row 2*oh0 - 3 + r, pixel
// j <-> image column j - 3; zero outside the image; channels >= c_in zeroed.
__device__ __forceinline__ void stem_stage_image(const StemParams &p, const StemItem &t, uint2 *img_s, int tid)
{
    const int RPX = stem_rpx(p.wo);
    const uint2 *img = reinterpret_cast<const uint2 *>(p.img);
    const uint32_t keep_lo = p.c_in >= 2 ? 0xffffffffu : 0x0000ffffu;
    const uint32_t keep_hi = p.c_in >= 4 ? 0xffffffffu : (p.c_in == 3 ? 0x0000ffffu : 0u);
    const int ih0 = 2 * t.oh0 - kStemPad;
    for (int q = tid; q < kSIR * RPX; q += kThreads) {
        const int r = q / RPX, j = q - r * RPX;
        const int ih = ih0 + r, iw = j - kStemPad;
        uint2 v = make_uint2(0u, 0u);
        if (ih >= 0 && ih < p.h && iw >= 0 && iw < p.w) {
            v = img[((int64_t)t.n * p.h + ih) * p.w + iw];
            v.x &= keep_lo;
            v.y &= keep_hi;
        }
        img_s[q] = v;
    }
}

}  // namespace

// --------------------------------------------------------------------------
// First CONV forward (bf16): out[n][oh][ow][co] = sum_{kh,kw,ci} img[n][2oh-3+kh]
// [2ow-3+kw][ci] w[kh][kw][ci][co], optional per-channel sum / sum of squares
// of the stored (bf16-rounded) outputs, one partial row per workgroup.
// Wave w computes the item's 16-pixel blocks w, w+4, ... for all 64 channels.
template <bool STATS>
__global__ __launch_bounds__(kThreads, 2) void k_stem_conv(StemParams p)
{
    using M = Mfma<bf16_t>;
    extern __shared__ __align__(16) unsigned char smem[];
    const int RPX = stem_rpx(p.wo);
    uint2 *img_s = reinterpret_cast<uint2 *>(smem);
    bf16_t *stg = reinterpret_cast<bf16_t *>(smem + (size_t)kSIR * RPX * 8);   // [4 waves][4][16][kSPitch]
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g16 = lane >> 4, l16 = lane & 15;
    const int wo = p.wo;
    const int MB = (kStemRows * wo + 15) / 16;
    const int64_t items = (int64_t)p.n * ((p.ho + kStemRows - 1) / kStemRows);

    // weight fragments: K step kh, lane k = 8*g16 + e <-> kw = 2*g16 + e/4, ci = e%4
    bf16x8 bw[kSK][4];
    const bf16_t *wt = reinterpret_cast<const bf16_t *>(p.wt);
    #pragma unroll
    for (int kh = 0; kh < kSK; kh++)
        #pragma unroll
        for (int nb = 0; nb < 4; nb++) {
            uint32_t wd[4];
            #pragma unroll
            for (int e2 = 0; e2 < 4; e2++) {
                uint32_t h2[2];
                #pragma unroll
                for (int u = 0; u < 2; u++) {
                    // (an unconditional load at a clamped index, then a select:
                    // a load under a branch costs one memory round trip each)
                    const int e = 2 * e2 + u, kw = 2 * g16 + e / 4, ci = e % 4;
                    const bool ok = kw < kSK && ci < p.c_in;
                    const uint32_t v =
                        wt[ok ? ((kh * kSK + kw) * p.c_in + ci) * kStemCout + nb * 16 + l16 : nb * 16 + l16];
                    h2[u] = ok ? v : 0u;
                }
                wd[e2] = h2[0] | (h2[1] << 16);
            }
            bw[kh][nb] = M::from_words(wd);
        }

    float s1[4] = {0.f, 0.f, 0.f, 0.f}, s2[4] = {0.f, 0.f, 0.f, 0.f}, sh[4] = {0.f, 0.f, 0.f, 0.f};
    if (STATS && p.shift)                         // statistics of s - shift
        for (int nb = 0; nb < 4; nb++) sh[nb] = p.shift[nb * 16 + (threadIdx.x & 15)];
    const int lid = xcd_remap(blockIdx.x, gridDim.x);
    for (int64_t it = lid; it < items; it += gridDim.x) {
        const StemItem t = stem_item(p, it);
        stem_stage_image(p, t, img_s, tid);
        __syncthreads();
        f32x4 acc[4][4];
        #pragma unroll
        for (int mi = 0; mi < 4; mi++)
            #pragma unroll
            for (int nb = 0; nb < 4; nb++) acc[mi][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
        #pragma unroll
        for (int mi = 0; mi < 4; mi++) {
            const int mb = wave + 4 * mi;
            if (mb < MB) {                                        // wave-uniform
                int pp = mb * 16 + l16;
                if (pp >= t.pv) pp = 0;                           // padding rows read pixel 0 (finite)
                const int r = pp / wo, ow = pp - r * wo;
                const bf16_t *a0 = reinterpret_cast<const bf16_t *>(img_s + 2 * r * RPX + 2 * ow + 2 * g16);
                #pragma unroll
                for (int kh = 0; kh < kSK; kh++) {
                    const bf16x8 a = M::load(a0 + (size_t)kh * RPX * 4);
                    #pragma unroll
                    for (int nb = 0; nb < 4; nb++) M::mma(acc[mi][nb], a, bw[kh][nb]);
                }
            }
        }
        // epilogue: round, statistics of the stored values, stage for coalesced stores
        #pragma unroll
        for (int mi = 0; mi < 4; mi++) {
            const int mb = wave + 4 * mi;
            if (mb < MB) {
                #pragma unroll
                for (int nb = 0; nb < 4; nb++)
                    #pragma unroll
                    for (int i = 0; i < 4; i++) {
                        const int pp = mb * 16 + 4 * g16 + i;
                        const bf16_t b = f2bf(acc[mi][nb][i]);
                        if (STATS && pp < t.pv) {
                            const float v = bf2f(b) - sh[nb];
                            s1[nb] += v;
                            s2[nb] += v * v;
                        }
                        stg[((wave * 4 + mi) * 16 + 4 * g16 + i) * kSPitch + nb * 16 + l16] = b;
                    }
            }
        }
        __syncthreads();
        bf16_t *dst = reinterpret_cast<bf16_t *>(p.s) + ((int64_t)t.n * p.ho + t.oh0) * wo * kStemCout;
        for (int v = tid; v < t.pv * 8; v += kThreads) {
            const int pp = v >> 3, c8 = v & 7, mb = pp >> 4;
            const bf16_t *src = stg + (((mb & 3) * 4 + (mb >> 2)) * 16 + (pp & 15)) * kSPitch + c8 * 8;
            stg16(dst + (int64_t)pp * kStemCout + c8 * 8, *reinterpret_cast<const vec16 *>(src));
        }
        __syncthreads();
    }
    if (STATS) {
        #pragma unroll
        for (int nb = 0; nb < 4; nb++) {
            s1[nb] += __shfl_xor(s1[nb], 16, 64);
            s1[nb] += __shfl_xor(s1[nb], 32, 64);
            s2[nb] += __shfl_xor(s2[nb], 16, 64);
            s2[nb] += __shfl_xor(s2[nb], 32, 64);
        }
        float *red = reinterpret_cast<float *>(stg);              // [4 waves][2][64]
        if (g16 == 0)
            #pragma unroll
            for (int nb = 0; nb < 4; nb++) {
                red[(wave * 2) * kStemCout + nb * 16 + l16] = s1[nb];
                red[(wave * 2 + 1) * kStemCout + nb * 16 + l16] = s2[nb];
            }
        __syncthreads();
        if (tid < 2 * kStemCout) {
            const int k = tid / kStemCout, c = tid - k * kStemCout;
            float a = 0.f;
            for (int wv = 0; wv < 4; wv++) a += red[(wv * 2 + k) * kStemCout + c];
            p.part[(int64_t)blockIdx.x * 2 * kStemCout + k * kStemCout + c] = a;
        }
    }
}

// float32 first CONV: one thread per output element (the float32
// configuration only runs at test sizes).
__global__ __launch_bounds__(kThreads) void k_stem_conv_f32(StemParams p)
{
    const float *img = reinterpret_cast<const float *>(p.img), *wt = reinterpret_cast<const float *>(p.wt);
    float *out = reinterpret_cast<float *>(p.s);
    const int64_t total = (int64_t)p.n * p.ho * p.wo * kStemCout;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < total; i += (int64_t)gridDim.x * kThreads) {
        const int co = (int)(i % kStemCout);
        const int64_t pix = i / kStemCout;
        const int ow = (int)(pix % p.wo);
        const int64_t t = pix / p.wo;
        const int oh = (int)(t % p.ho);
        const int64_t n = t / p.ho;
        float acc = 0.f;
        for (int kh = 0; kh < kSK; kh++) {
            const int ih = 2 * oh - kStemPad + kh;
            if (ih < 0 || ih >= p.h) continue;
            for (int kw = 0; kw < kSK; kw++) {
                const int iw = 2 * ow - kStemPad + kw;
                if (iw < 0 || iw >= p.w) continue;
                const float *x = img + ((n * p.h + ih) * p.w + iw) * kStemPix;
                for (int ci = 0; ci < p.c_in; ci++)
                    acc = __builtin_fmaf(x[ci], wt[((kh * kSK + kw) * p.c_in + ci) * kStemCout + co], acc);
            }
        }
        out[i] = acc;
    }
}

// --------------------------------------------------------------------------
// First CONV weight gradient (bf16): dW[kh][kw][ci][co] = sum over output
// pixels of img(patch) * g, g the gradient of the CONV output (dense, or the
// deferred input gradient of the BN after it, formed on load and rounded to
// bf16 as a materialised gradient would be).  Split-K over items: each
// workgroup writes one float32 partial of dW.  Both operands are staged
// row-major and read transposed (ds_read_b64_tr_b16): the G rows are output
// pixels x 64 channels; the patch row of pixel p for filter row kh is the 32
// elements at pixel 2*ow of staged input row kh + 2r.  Wave w owns the
// 16-wide k blocks w, w+4, ... (k = kh*32 + kw*4 + ci) for all 64 channels.
typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4_t lds_s16x4_t;

__device__ __forceinline__ bf16x8 tr_pair(const bf16_t *lo, const bf16_t *hi)
{
    const s16x4_t a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t *)(lo));
    const s16x4_t b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t *)(hi));
    typedef short s16x8_t __attribute__((ext_vector_type(8)));
    const s16x8_t v = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
    return __builtin_bit_cast(bf16x8, v);
}

template <int GS>
__global__ __launch_bounds__(kThreads, 2) void k_stem_wgrad(StemParams p)
{
    using M = Mfma<bf16_t>;
    extern __shared__ __align__(16) unsigned char smem[];
    const int RPX = stem_rpx(p.wo);
    const int wo = p.wo;
    const int PP = (kStemRows * wo + 31) / 32 * 32;
    uint2 *img_s = reinterpret_cast<uint2 *>(smem);
    bf16_t *Gs = reinterpret_cast<bf16_t *>(smem + (size_t)kSIR * RPX * 8);   // [PP][kSPitch]
    float *gco = reinterpret_cast<float *>(Gs + (size_t)PP * kSPitch);         // [3][64]
    const bf16_t *img_e = reinterpret_cast<const bf16_t *>(img_s);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g16 = lane >> 4, l16 = lane & 15;
    const int64_t m_out = (int64_t)p.n * p.ho * wo;
    const int64_t items = (int64_t)p.n * ((p.ho + kStemRows - 1) / kStemRows);

    if (GS == GB_BNGRAD && tid < kStemCout) {
        float A, B, C;
        deferred_coef(0, tid, 1.0f / (float)m_out, p.g_gamma, p.g_mean, p.g_rstd, p.g_dgamma, p.g_dbeta, nullptr,
                      nullptr, A, B, C);
        gco[tid] = A;
        gco[kStemCout + tid] = B;
        gco[2 * kStemCout + tid] = C;
    }
    __syncthreads();

    f32x4 acc[4][4];
    #pragma unroll
    for (int ki = 0; ki < 4; ki++)
        #pragma unroll
        for (int cb = 0; cb < 4; cb++) acc[ki][cb] = f32x4{0.f, 0.f, 0.f, 0.f};

    const bf16_t *gsrc = reinterpret_cast<const bf16_t *>(p.g);
    const bf16_t *gx = reinterpret_cast<const bf16_t *>(p.gx);
    for (int64_t it = blockIdx.x; it < items; it += gridDim.x) {
        const StemItem t = stem_item(p, it);
        stem_stage_image(p, t, img_s, tid);
        const int64_t q0 = ((int64_t)t.n * p.ho + t.oh0) * wo;
        for (int v = tid; v < PP * 8; v += kThreads) {
            const int pp = v >> 3, c8 = v & 7;
            vec16 o = zero16();
            if (pp < t.pv) {
                const int64_t q = q0 + pp;
                if (GS == GB_BNGRAD) {
                    float d[8], x[8];
                    Elem<bf16_t>::unpack(ldg16(gsrc + q * kStemCout + c8 * 8), d);
                    Elem<bf16_t>::unpack(ldg16(gx + q * p.gx_ldc + c8 * 8), x);
                    #pragma unroll
                    for (int e = 0; e < 8; e++) {
                        const int c = c8 * 8 + e;
                        d[e] = __builtin_fmaf(gco[c], d[e], __builtin_fmaf(gco[kStemCout + c], x[e],
                                                                            gco[2 * kStemCout + c]));
                    }
                    o = Elem<bf16_t>::pack(d);
                } else {
                    o = ldg16(gsrc + q * p.g_ldc + c8 * 8);
                }
            }
            *reinterpret_cast<vec16 *>(Gs + pp * kSPitch + c8 * 8) = o;
        }
        __syncthreads();
        for (int p0 = 0; p0 < PP; p0 += 32) {
            bf16x8 b[4];
            const bf16_t *gb = Gs + (p0 + 8 * g16 + (l16 >> 2)) * kSPitch + 4 * (l16 & 3);
            #pragma unroll
            for (int cb = 0; cb < 4; cb++) b[cb] = tr_pair(gb + cb * 16, gb + 4 * kSPitch + cb * 16);
            // patch rows of this lane's two pixels (padding pixels read pixel 0)
            int plo = p0 + 8 * g16 + (l16 >> 2), phi = plo + 4;
            if (plo >= t.pv) plo = 0;
            if (phi >= t.pv) phi = 0;
            const int rlo = plo / wo, rhi = phi / wo;
            const int blo = 2 * rlo * RPX + 2 * (plo - rlo * wo) + (l16 & 3);
            const int bhi = 2 * rhi * RPX + 2 * (phi - rhi * wo) + (l16 & 3);
            #pragma unroll
            for (int ki = 0; ki < 4; ki++) {
                const int kb = wave + 4 * ki;
                if (kb < kSKB) {                                   // wave-uniform
                    const int off = ((kb >> 1) * RPX + 4 * (kb & 1)) * 4;
                    const bf16x8 a = tr_pair(img_e + (size_t)blo * 4 + off, img_e + (size_t)bhi * 4 + off);
                    #pragma unroll
                    for (int cb = 0; cb < 4; cb++) M::mma(acc[ki][cb], a, b[cb]);
                }
            }
        }
        __syncthreads();
    }
    // partial dW: C row k = kb*16 + 4*g16 + i <-> kh = kb/2, kw = 4*(kb%2) + g16, ci = i
    float *dst = p.dwpart + (int64_t)blockIdx.x * kSK * kSK * p.c_in * kStemCout;
    #pragma unroll
    for (int ki = 0; ki < 4; ki++) {
        const int kb = wave + 4 * ki;
        if (kb >= kSKB) continue;
        const int kh = kb >> 1, kw = 4 * (kb & 1) + g16;
        if (kw >= kSK) continue;
        #pragma unroll
        for (int cb = 0; cb < 4; cb++)
            #pragma unroll
            for (int i = 0; i < 4; i++)
                if (i < p.c_in) dst[((kh * kSK + kw) * p.c_in + i) * kStemCout + cb * 16 + l16] = acc[ki][cb][i];
    }
}

// float32 first-CONV weight gradient: one thread per weight, summing over all
// output pixels (test sizes).
template <int GS>
__global__ __launch_bounds__(kThreads) void k_stem_wgrad_f32(StemParams p)
{
    const int nw = kSK * kSK * p.c_in * kStemCout;
    const int i = blockIdx.x * kThreads + threadIdx.x;
    if (i >= nw) return;
    const int co = i % kStemCout, r = i / kStemCout;
    const int ci = r % p.c_in, kw = (r / p.c_in) % kSK, kh = r / (p.c_in * kSK);
    const int64_t m_out = (int64_t)p.n * p.ho * p.wo;
    float A = 1.f, B = 0.f, C = 0.f, K = 0.f;
    if (GS == GB_BNGRAD) {
        deferred_coef(0, co, 1.0f / (float)m_out, p.g_gamma, p.g_mean, p.g_rstd, p.g_dgamma, p.g_dbeta, nullptr,
                      nullptr, A, B, C);
        K = bn_centre<float>(p.g_ctr, co);      // d = A dy + B (x - K) + C
    }
    const float *img = reinterpret_cast<const float *>(p.img);
    const float *g = reinterpret_cast<const float *>(p.g), *gx = reinterpret_cast<const float *>(p.gx);
    float acc = 0.f;
    for (int64_t q = 0; q < m_out; q++) {
        const int ow = (int)(q % p.wo);
        const int64_t t = q / p.wo;
        const int oh = (int)(t % p.ho);
        const int64_t n = t / p.ho;
        const int ih = 2 * oh - kStemPad + kh, iw = 2 * ow - kStemPad + kw;
        if (ih < 0 || ih >= p.h || iw < 0 || iw >= p.w) continue;
        const float gv = GS == GB_BNGRAD ? __builtin_fmaf(A, g[q * kStemCout + co], __builtin_fmaf(B, gx[q * p.gx_ldc + co] - K, C))
                                         : g[q * p.g_ldc + co];
        acc = __builtin_fmaf(img[((n * p.h + ih) * p.w + iw) * kStemPix + ci], gv, acc);
    }
    p.dwpart[i] = acc;
}

// --------------------------------------------------------------------------
// 3x3 / stride 2 / pad 1 max pooling (taps outside the image never win), with
// BN: y = relu(gamma*(x-mean)*rstd + beta) pooled.  The transform is monotone
// per channel (increasing for gamma > 0, decreasing for gamma < 0, constant
// for gamma = 0), so the first maximum of the transformed window is the first
// maximum of sign(gamma)*x (for gamma = 0 the first tap), and the pooled value
// is the transform of the input there.  Without BN: plain max pooling of x.
// STATS: per-channel sum and sum of squares of the stored outputs.  Row
// blocks over output pixels as in the statistics sweeps.
template <typename T, bool BN, bool STATS>
__global__ __launch_bounds__(kThreads) void k_maxpool_fwd(MaxPoolParams p, int64_t rows_per_block)
{
    constexpr int VEC = Elem<T>::VEC;
    __shared__ float red[2][STATS ? kThreads * VEC : 1];
    const int C = p.c, ho = p.ho, wo = p.wo;
    const int64_t m_out = (int64_t)p.n * ho * wo;
    const int cvec = C / VEC;
    const int vb = min(kStatsMaxVec, cvec - (int)blockIdx.y * kStatsMaxVec);
    const int ry = kThreads / vb;
    const int tid = threadIdx.x, tx = tid % vb, ty = tid / vb;
    const int c0 = ((int)blockIdx.y * kStatsMaxVec + tx) * VEC;
    float sg[VEC], k[VEC], b[VEC], kc[VEC], s1[VEC], s2[VEC], sh[VEC];
    #pragma unroll
    for (int i = 0; i < VEC; i++) { s1[i] = s2[i] = 0.f; sh[i] = 0.f; sg[i] = 1.f; k[i] = 1.f; b[i] = 0.f; kc[i] = 0.f; }
    if (STATS && p.shift && ty < ry)                                      // statistics of y - shift
        #pragma unroll
        for (int i = 0; i < VEC; i++) sh[i] = p.shift[c0 + i];
    if (BN && ty < ry) {            // (all loads in one branch: one memory round trip)
        float g[VEC], be[VEC], mu[VEC], rs[VEC];
        #pragma unroll
        for (int i = 0; i < VEC; i++) {
            g[i] = p.gamma[c0 + i]; be[i] = p.beta[c0 + i]; mu[i] = p.mean[c0 + i]; rs[i] = p.rstd[c0 + i];
            kc[i] = bn_centre<T>(p.ctr, c0 + i);
        }
        #pragma unroll
        for (int i = 0; i < VEC; i++) {
            sg[i] = g[i] > 0.f ? 1.f : (g[i] < 0.f ? -1.f : 0.f);
            bn_coef(g[i], be[i], mu[i], rs[i], k[i], b[i]);
        }
    }
    const T *x = reinterpret_cast<const T *>(p.x);
    T *y = reinterpret_cast<T *>(p.y);
    const int64_t r0 = (int64_t)blockIdx.x * rows_per_block;
    const int64_t r1 = min(m_out, r0 + rows_per_block);
    if (ty < ry) {
        for (int64_t r = r0 + ty; r < r1; r += ry) {
            const int ow = (int)(r % wo);
            const int64_t t = r / wo;
            const int oh = (int)(t % ho);
            const int64_t n = t / ho;
            float best[VEC], bv[VEC];
            #pragma unroll
            for (int i = 0; i < VEC; i++) { best[i] = -INFINITY; bv[i] = 0.f; }
            // the nine taps' loads first, at clamped positions (a load under a
            // bounds branch costs one memory round trip each), then the
            // first-maximum scan in tap order over the taps inside the image
            vec16 tv[9];
            bool tin[9];
            #pragma unroll
            for (int t9 = 0; t9 < 9; t9++) {
                const int ih = 2 * oh - 1 + t9 / 3, iw = 2 * ow - 1 + t9 % 3;
                tin[t9] = ih >= 0 && ih < p.h && iw >= 0 && iw < p.w;
                const int ihc = ih < 0 ? 0 : (ih >= p.h ? p.h - 1 : ih), iwc = iw < 0 ? 0 : (iw >= p.w ? p.w - 1 : iw);
                tv[t9] = ldg16(x + ((n * p.h + ihc) * p.w + iwc) * p.x_ldc + c0);
            }
            #pragma unroll
            for (int t9 = 0; t9 < 9; t9++) {
                if (!tin[t9]) continue;
                float f[VEC];
                Elem<T>::unpack(tv[t9], f);
                #pragma unroll
                for (int i = 0; i < VEC; i++) {
                    const float key = BN ? sg[i] * f[i] : f[i];
                    if (key > best[i]) { best[i] = key; bv[i] = f[i]; }
                }
            }
            float o[VEC];
            #pragma unroll
            for (int i = 0; i < VEC; i++) {
                o[i] = bv[i];
                if (BN) {
                    const float v = bn_lin(bv[i] - kc[i], k[i], b[i]);
                    o[i] = v > 0.f ? v : 0.f;
                }
            }
            const vec16 ov = Elem<T>::pack(o);
            stg16(y + r * p.y_ldc + c0, ov);
            if (STATS) {
                Elem<T>::unpack(ov, o);
                #pragma unroll
                for (int i = 0; i < VEC; i++) { const float d = o[i] - sh[i]; s1[i] += d; s2[i] += d * d; }
            }
        }
    }
    if (STATS) {
        const int nch = vb * VEC;
        if (ty < ry)
            #pragma unroll
            for (int i = 0; i < VEC; i++) {
                red[0][ty * nch + tx * VEC + i] = s1[i];
                red[1][ty * nch + tx * VEC + i] = s2[i];
            }
        __syncthreads();
        if (tid < nch) {
            float a = 0.f, bb = 0.f;
            for (int j = 0; j < ry; j++) { a += red[0][j * nch + tid]; bb += red[1][j * nch + tid]; }
            const int c = (int)blockIdx.y * kStatsMaxVec * VEC + tid;
            float *pr = p.part + (int64_t)blockIdx.x * 2 * C;
            pr[c] = a;
            pr[C + c] = bb;
        }
    }
}

// Backward of k_maxpool_fwd.  Item = (image, input rows 2j and 2j+1), whose
// pooling windows are those of output rows j and j+1.  Phase 1 writes, per
// window of those two output rows and channel, the tap index of its first
// maximum (as in the forward pass) to LDS; phase 2 gives every input pixel of
// the two rows the sum of the gradients of the windows (in row-major window
// order) whose maximum it is.  With BN the result dz is the gradient of the
// ReLU output: dy = dz [y > 0] (y recomputed from x) is stored and the BN
// reductions sum(dy), sum(dy * xhat) of the stored dy are accumulated; without
// BN dz is stored.  The per-thread channel vector is fixed (256 is a multiple
// of the vectors per pixel), so the sums stay in registers across items.
template <typename T, bool BN>
__global__ __launch_bounds__(kThreads) void k_maxpool_bwd(MaxPoolParams p)
{
    constexpr int VEC = Elem<T>::VEC;
    __shared__ __align__(16) uint8_t codes[2][kMaxPoolMaxWo * kMaxPoolMaxC];
    __shared__ float red[2][BN ? kThreads * VEC : 1];
    __shared__ float sgn_s[kMaxPoolMaxC];                         // sign(gamma) per channel
    const int C = p.c, h = p.h, w = p.w, ho = p.ho, wo = p.wo;
    const int cvec = C / VEC;
    const int tid = threadIdx.x, cv = tid % cvec;
    const int hp = (h + 1) / 2;
    const int64_t items = (int64_t)p.n * hp;
    float k[VEC], b[VEC], mu[VEC], rs[VEC], kc[VEC], s1[VEC], s2[VEC];
    #pragma unroll
    for (int i = 0; i < VEC; i++) {
        s1[i] = s2[i] = 0.f;
        k[i] = 1.f; b[i] = 0.f; mu[i] = 0.f; rs[i] = 1.f; kc[i] = 0.f;
        if (BN) {
            const int c = cv * VEC + i;
            const float g = p.gamma[c];
            mu[i] = p.mean[c];
            rs[i] = p.rstd[c];
            kc[i] = bn_centre<T>(p.ctr, c);
            bn_coef(g, p.beta[c], mu[i], rs[i], k[i], b[i]);
        }
    }
    if (BN && tid < C) {
        const float g = p.gamma[tid];
        sgn_s[tid] = g > 0.f ? 1.f : (g < 0.f ? -1.f : 0.f);
    }
    __syncthreads();
    const T *x = reinterpret_cast<const T *>(p.x);
    const T *gy = reinterpret_cast<const T *>(p.g);
    T *dy = reinterpret_cast<T *>(p.y);
    for (int64_t it = blockIdx.x; it < items; it += gridDim.x) {
        const int64_t n = it / hp;
        const int j = (int)(it - n * hp);
        // phase 1: first-maximum taps of output rows j, j + 1
        for (int t = tid; t < 2 * wo * cvec; t += kThreads) {
            const int orow = t / (wo * cvec), rem = t - orow * wo * cvec;
            const int ow = rem / cvec, v = rem - ow * cvec;
            const int oh = j + orow;
            if (oh >= ho) continue;
            float best[VEC];
            uint32_t code[VEC];
            #pragma unroll
            for (int i = 0; i < VEC; i++) { best[i] = -INFINITY; code[i] = 0; }
            // the nine taps' loads first at clamped positions, then the scan
            // in tap order (as in the forward pass)
            vec16 tv[9];
            bool tin[9];
            #pragma unroll
            for (int t9 = 0; t9 < 9; t9++) {
                const int ih = 2 * oh - 1 + t9 / 3, iw = 2 * ow - 1 + t9 % 3;
                tin[t9] = ih >= 0 && ih < h && iw >= 0 && iw < w;
                const int ihc = ih < 0 ? 0 : (ih >= h ? h - 1 : ih), iwc = iw < 0 ? 0 : (iw >= w ? w - 1 : iw);
                tv[t9] = ldg16(x + ((n * h + ihc) * w + iwc) * p.x_ldc + v * VEC);
            }
            #pragma unroll
            for (int t9 = 0; t9 < 9; t9++) {
                if (!tin[t9]) continue;
                float f[VEC];
                Elem<T>::unpack(tv[t9], f);
                #pragma unroll
                for (int i = 0; i < VEC; i++) {
                    const float kk = BN ? sgn_s[v * VEC + i] * f[i] : f[i];
                    if (kk > best[i]) { best[i] = kk; code[i] = (uint32_t)t9; }
                }
            }
            uint8_t *cp = &codes[orow][ow * C + v * VEC];
            #pragma unroll
            for (int i = 0; i < VEC; i++) cp[i] = (uint8_t)code[i];
        }
        __syncthreads();
        // phase 2: input rows 2j, 2j + 1
        for (int t = tid; t < 2 * w * cvec; t += kThreads) {
            const int ir = t / (w * cvec), col = (t - ir * w * cvec) / cvec;
            const int row = 2 * j + ir;
            if (row >= h) continue;
            float dz[VEC];
            #pragma unroll
            for (int i = 0; i < VEC; i++) dz[i] = 0.f;
            const int oh_lo = j, oh_hi = ir ? j + 1 : j;
            const int ow_lo = col >> 1, ow_hi = (col & 1) ? (col + 1) >> 1 : col >> 1;
            // the (at most 2 x 2) covering windows' gradients and the BN input
            // loaded first at clamped positions, then summed in row-major
            // window order
            const int64_t q = (n * h + row) * w + col;
            vec16 gv[4], xv = zero16();
            bool win[4];
            #pragma unroll
            for (int w4 = 0; w4 < 4; w4++) {
                const int oh = oh_lo + (w4 >> 1), ow = ow_lo + (w4 & 1);
                win[w4] = oh <= oh_hi && oh < ho && ow <= ow_hi && ow < wo;
                const int ohc = oh < ho ? oh : ho - 1, owc = ow < wo ? ow : wo - 1;
                gv[w4] = ldg16(gy + ((n * ho + ohc) * wo + owc) * p.g_ldc + cv * VEC);
            }
            if (BN) xv = ldg16(x + q * p.x_ldc + cv * VEC);
            #pragma unroll
            for (int w4 = 0; w4 < 4; w4++) {
                if (!win[w4]) continue;
                const int oh = oh_lo + (w4 >> 1), ow = ow_lo + (w4 & 1);
                const uint32_t tap = (uint32_t)((row - (2 * oh - 1)) * 3 + (col - (2 * ow - 1)));
                float g[VEC];
                Elem<T>::unpack(gv[w4], g);
                const uint8_t *cp = &codes[oh - j][ow * C + cv * VEC];
                #pragma unroll
                for (int i = 0; i < VEC; i++)
                    if (cp[i] == tap) dz[i] += g[i];
            }
            float o[VEC];
            if (BN) {
                float f[VEC];
                Elem<T>::unpack(xv, f);
                #pragma unroll
                for (int i = 0; i < VEC; i++) o[i] = bn_lin(f[i] - kc[i], k[i], b[i]) > 0.f ? dz[i] : 0.f;
                const vec16 ov = Elem<T>::pack(o);
                stg16(dy + q * C + cv * VEC, ov);
                Elem<T>::unpack(ov, o);
                #pragma unroll
                for (int i = 0; i < VEC; i++) {
                    s1[i] += o[i];
                    s2[i] += o[i] * (((f[i] - kc[i]) - mu[i]) * rs[i]);
                }
            } else {
                stg16(dy + q * C + cv * VEC, Elem<T>::pack(dz));
            }
        }
        __syncthreads();
    }
    if (BN) {
        // threads tid = cv + cvec*u hold channel vector cv
        #pragma unroll
        for (int i = 0; i < VEC; i++) {
            red[0][tid * VEC + i] = s1[i];
            red[1][tid * VEC + i] = s2[i];
        }
        __syncthreads();
        if (tid < C) {
            const int v = tid / VEC, i = tid - v * VEC;
            float a = 0.f, bb = 0.f;
            for (int u = v; u < kThreads; u += cvec) { a += red[0][u * VEC + i]; bb += red[1][u * VEC + i]; }
            float *pr = p.part + (int64_t)blockIdx.x * 2 * C;
            pr[tid] = a;
            pr[C + tid] = bb;
        }
    }
}

// --------------------------------------------------------------------------
// Classifier head.
// Global average pooling of relu(bn(x)): f[n][c] = (1/hw) sum_p relu(...),
// one thread per (image, channel vector), pixels summed in order.
template <typename T>
__global__ __launch_bounds__(kThreads) void k_head_pool(HeadParams p)
{
    constexpr int VEC = Elem<T>::VEC;
    const int cvec = p.c / VEC, hw = p.h * p.w;
    const int i = blockIdx.x * kThreads + threadIdx.x;
    if (i >= p.n * cvec) return;
    const int n = i / cvec, c0 = (i - n * cvec) * VEC;
    float k[VEC], b[VEC], kc[VEC], acc[VEC];
    #pragma unroll
    for (int e = 0; e < VEC; e++) {
        bn_coef(p.gamma[c0 + e], p.beta[c0 + e], p.mean[c0 + e], p.rstd[c0 + e], k[e], b[e]);
        kc[e] = bn_centre<T>(p.ctr, c0 + e);
        acc[e] = 0.f;
    }
    const T *x = reinterpret_cast<const T *>(p.x);
    for (int q = 0; q < hw; q++) {
        float f[VEC];
        Elem<T>::unpack(ldg16(x + ((int64_t)n * hw + q) * p.x_ldc + c0), f);
        #pragma unroll
        for (int e = 0; e < VEC; e++) {
            const float v = bn_lin(f[e] - kc[e], k[e], b[e]);
            acc[e] += v > 0.f ? v : 0.f;
        }
    }
    const float inv = 1.0f / (float)hw;
    #pragma unroll
    for (int e = 0; e < VEC; e++) p.f[(int64_t)n * p.c + c0 + e] = acc[e] * inv;
}

// Small float32 GEMM for the FC layer: out[i][j] = sum_k A(i,k) B(k,j) (+ bias[j]),
// A(i,k) = a[i*sai + k*sak] (float32), B(k,j) = b[k*sbk + j*sbj] (TB).  16 x
// kFcBN output tiles (for the 128-image batch: 8 x 63 workgroups, two per CU
// and more), K in chunks of 64 staged in LDS with the operand's contiguous
// index running across the threads (coalesced for either orientation),
// kFcBN / 16 consecutive outputs of one row per thread (A staged [i][k]: four
// k of its row in one 16-byte LDS read), k summed in order (deterministic).
constexpr int kFcBN = 16;                 // output columns per workgroup tile
template <typename TB>
__global__ __launch_bounds__(kThreads) void k_fc_gemm(int M, int N, int K, const float *__restrict__ a, int64_t sai,
                                                      int64_t sak, const TB *__restrict__ b, int64_t sbk,
                                                      int64_t sbj, const float *__restrict__ bias,
                                                      float *__restrict__ out)
{
    constexpr int BM = 16, BN = kFcBN, BK = 64;
    __shared__ __align__(16) float As[BM][BK + 4];
    __shared__ __align__(16) float Bs[BK][BN + 4];
    const int tid = threadIdx.x, tr = tid / 16, tc = tid % 16;
    const int i0 = blockIdx.y * BM, j0 = blockIdx.x * BN;
    constexpr int OPT = BN / 16;                     // consecutive outputs per thread
    float acc[OPT];
    #pragma unroll
    for (int v = 0; v < OPT; v++) acc[v] = 0.f;
    constexpr int NA = BK * BM / kThreads, NB = BK * BN / kThreads;
    for (int k0 = 0; k0 < K; k0 += BK) {
        // every load of the chunk at a clamped index first, then the LDS
        // writes with the out-of-range elements selected to zero (a load
        // under a bounds branch costs one memory round trip each)
        float av[NA];
        TB bv[NB];                                   // raw: converted after every load is issued
        bool aok[NA], bok[NB];
        #pragma unroll
        for (int u = 0; u < NA; u++) {
            const int e = tid + u * kThreads;
            const int kk = sak == 1 ? e % BK : e / BM, ii = sak == 1 ? e / BK : e % BM;
            const int gi = i0 + ii, gk = k0 + kk;
            aok[u] = gi < M && gk < K;
            av[u] = a[(aok[u] ? gi : 0) * sai + (aok[u] ? gk : 0) * sak];
        }
        #pragma unroll
        for (int u = 0; u < NB; u++) {
            const int e = tid + u * kThreads;
            const int kk = sbk == 1 ? e % BK : e / BN, jj = sbk == 1 ? e / BK : e % BN;
            const int gj = j0 + jj, gk = k0 + kk;
            bok[u] = gj < N && gk < K;
            const int64_t off = (int64_t)(bok[u] ? gk : 0) * sbk + (int64_t)(bok[u] ? gj : 0) * sbj;
            bv[u] = b[off];
        }
        __builtin_amdgcn_sched_barrier(0);   // keep every load above the writes (the scheduler sinks them)
        #pragma unroll
        for (int u = 0; u < NA; u++) {
            const int e = tid + u * kThreads;
            const int kk = sak == 1 ? e % BK : e / BM, ii = sak == 1 ? e / BK : e % BM;
            As[ii][kk] = aok[u] ? av[u] : 0.f;
        }
        #pragma unroll
        for (int u = 0; u < NB; u++) {
            const int e = tid + u * kThreads;
            const int kk = sbk == 1 ? e % BK : e / BN, jj = sbk == 1 ? e / BK : e % BN;
            float f;
            if constexpr (sizeof(TB) == 2) f = bf2f(bv[u]);
            else f = bv[u];
            Bs[kk][jj] = bok[u] ? f : 0.f;
        }
        __syncthreads();
        #pragma unroll 4
        for (int k4 = 0; k4 < BK; k4 += 4) {
            const float4 a4 = *reinterpret_cast<const float4 *>(&As[tr][k4]);
            const float ak[4] = {a4.x, a4.y, a4.z, a4.w};
            #pragma unroll
            for (int q = 0; q < 4; q++) {
                #pragma unroll
                for (int v = 0; v < OPT; v++) acc[v] = __builtin_fmaf(ak[q], Bs[k4 + q][OPT * tc + v], acc[v]);
            }
        }
        __syncthreads();
    }
    #pragma unroll
    for (int v = 0; v < OPT; v++) {
        const int gi = i0 + tr, gj = j0 + OPT * tc + v;
        if (gi < M && gj < N) out[(int64_t)gi * N + gj] = acc[v] + (bias ? bias[gj] : 0.f);
    }
}

// Softmax cross-entropy of logits [n][K] against labels and its gradient
// dlogits = (softmax - onehot) / n: one workgroup per row, which writes the
// row's loss to loss[1 + r]; k_loss_mean then adds the rows in order
// (deterministic) into loss[0].  A label outside [0, K) gives a NaN loss.
__global__ __launch_bounds__(kThreads) void k_softmax_ce(int n, int K, const float *__restrict__ logits,
                                                         const int32_t *__restrict__ labels,
                                                         float *__restrict__ dlogits, float *__restrict__ loss)
{
    __shared__ float red[kThreads / 64];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int r = blockIdx.x;
    const float *z = logits + (int64_t)r * K;
    float mx = -INFINITY;
    for (int j = tid; j < K; j += kThreads) mx = fmaxf(mx, z[j]);
    for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
    if (lane == 0) red[wave] = mx;
    __syncthreads();
    mx = red[0];
    for (int w = 1; w < kThreads / 64; w++) mx = fmaxf(mx, red[w]);
    __syncthreads();
    float se = 0.f;
    for (int j = tid; j < K; j += kThreads) se += expf(z[j] - mx);
    se = wave_sum(se);
    if (lane == 0) red[wave] = se;
    __syncthreads();
    se = red[0];
    for (int w = 1; w < kThreads / 64; w++) se += red[w];
    const int lab = labels[r];
    const bool ok = lab >= 0 && lab < K;
    const float inv = 1.0f / se, invn = 1.0f / (float)n;
    for (int j = tid; j < K; j += kThreads)
        dlogits[(int64_t)r * K + j] = (expf(z[j] - mx) * inv - (j == lab ? 1.f : 0.f)) * invn;
    if (tid == 0) loss[1 + r] = ok ? logf(se) + mx - z[lab] : NAN;
}

__global__ __launch_bounds__(64) void k_loss_mean(int n, float *__restrict__ loss)
{
    if (threadIdx.x != 0) return;
    double t = 0.0;
    for (int r = 0; r < n; r++) t += (double)loss[1 + r];
    loss[0] = (float)(t / (double)n);
}

// db[j] = sum_n dlogits[n][j] (rows in order).
__global__ __launch_bounds__(kThreads) void k_colsum(int n, int K, const float *__restrict__ g, float *__restrict__ out)
{
    const int j = blockIdx.x * kThreads + threadIdx.x;
    if (j >= K) return;
    float s = 0.f;
    for (int r = 0; r < n; r++) s += g[(int64_t)r * K + j];
    out[j] = s;
}

// Head BN backward over x [m][c] (m = n*h*w): dz = df[n][c] / hw, y recomputed,
// dy = dz [y > 0] (float32, not stored);
//   HB_SPLIT: out = gamma*rstd*dy (the summed-gradient term of the BN) and the
//             partial sums of dy and dy*xhat;
//   HB_SUMS : the partial sums only;
//   HB_DX   : out = gamma*rstd*(dy - dbeta/m - xhat*dgamma/m) (dbeta, dgamma
//             from a previous HB_SUMS pass and its combine).
template <typename T, int MODE>
__global__ __launch_bounds__(kThreads) void k_head_bn_bwd(HeadParams p, int64_t rows_per_block)
{
    constexpr int VEC = Elem<T>::VEC;
    __shared__ float red[2][MODE == HB_DX ? 1 : kThreads * VEC];
    const int C = p.c, hw = p.h * p.w;
    const int64_t m = (int64_t)p.n * hw;
    const int cvec = C / VEC;
    const int vb = min(kStatsMaxVec, cvec - (int)blockIdx.y * kStatsMaxVec);
    const int ry = kThreads / vb;
    const int tid = threadIdx.x, tx = tid % vb, ty = tid / vb;
    const int c0 = ((int)blockIdx.y * kStatsMaxVec + tx) * VEC;
    float k[VEC], b[VEC], mu[VEC], rs[VEC], kc[VEC], gk[VEC], s1[VEC], s2[VEC], da[VEC], db[VEC];
    const float inv_hw = 1.0f / (float)hw, inv_m = 1.0f / (float)m;
    #pragma unroll
    for (int i = 0; i < VEC; i++) {
        s1[i] = s2[i] = 0.f;
        k[i] = b[i] = mu[i] = gk[i] = da[i] = db[i] = kc[i] = 0.f;
        rs[i] = 1.f;
    }
    if (ty < ry) {                  // (all loads in one branch: one memory round trip)
        float g[VEC], be[VEC];
        #pragma unroll
        for (int i = 0; i < VEC; i++) {
            const int c = c0 + i;
            mu[i] = p.mean[c]; rs[i] = p.rstd[c]; g[i] = p.gamma[c]; be[i] = p.beta[c];
            kc[i] = bn_centre<T>(p.ctr, c);
            if (MODE == HB_DX) { da[i] = p.dbeta[c]; db[i] = p.dgamma[c]; }
        }
        #pragma unroll
        for (int i = 0; i < VEC; i++) {
            bn_coef(g[i], be[i], mu[i], rs[i], k[i], b[i]);
            gk[i] = k[i];
            if (MODE == HB_DX) { da[i] *= inv_m; db[i] *= inv_m; }
        }
    }
    const T *x = reinterpret_cast<const T *>(p.x);
    T *out = reinterpret_cast<T *>(p.gx);
    const int64_t r0 = (int64_t)blockIdx.x * rows_per_block;
    const int64_t r1 = min(m, r0 + rows_per_block);
    if (ty < ry) {
        for (int64_t r = r0 + ty; r < r1; r += ry) {
            const int64_t n = r / hw;
            float f[VEC], o[VEC];
            Elem<T>::unpack(ldg16(x + r * p.x_ldc + c0), f);
            #pragma unroll
            for (int i = 0; i < VEC; i++) {
                const float dz = p.df[n * C + c0 + i] * inv_hw;
                const float xc = f[i] - kc[i];
                const float dyv = bn_lin(xc, k[i], b[i]) > 0.f ? dz : 0.f;
                const float xh = (xc - mu[i]) * rs[i];
                if (MODE == HB_DX) {
                    o[i] = gk[i] * (dyv - da[i] - xh * db[i]);
                } else {
                    o[i] = gk[i] * dyv;
                    s1[i] += dyv;
                    s2[i] += dyv * xh;
                }
            }
            if (MODE != HB_SUMS) stg16(out + r * p.gx_ldc + c0, Elem<T>::pack(o));
        }
    }
    if (MODE != HB_DX) {
        const int nch = vb * VEC;
        if (ty < ry)
            #pragma unroll
            for (int i = 0; i < VEC; i++) {
                red[0][ty * nch + tx * VEC + i] = s1[i];
                red[1][ty * nch + tx * VEC + i] = s2[i];
            }
        __syncthreads();
        if (tid < nch) {
            float a = 0.f, bb = 0.f;
            for (int j = 0; j < ry; j++) { a += red[0][j * nch + tid]; bb += red[1][j * nch + tid]; }
            const int c = (int)blockIdx.y * kStatsMaxVec * VEC + tid;
            float *pr = p.part + (int64_t)blockIdx.x * 2 * C;
            pr[c] = a;
            pr[C + c] = bb;
        }
    }
}

// --------------------------------------------------------------- launchers --
int64_t stem_groups(int64_t items) { return items < kStemMaxGroups ? (items < 1 ? 1 : items) : kStemMaxGroups; }

static size_t stem_lds(int wo, bool wgrad)
{
    const size_t img = (size_t)kSIR * stem_rpx(wo) * 8;
    if (!wgrad) return img + (size_t)4 * 4 * 16 * kSPitch * 2;
    const size_t PP = (size_t)(kStemRows * wo + 31) / 32 * 32;
    return img + PP * kSPitch * 2 + 3 * kStemCout * sizeof(float);
}

hipError_t launch_stem_conv(int dtype, const StemParams &p, bool stats, hipStream_t s)
{
    if (!p.img || !p.wt || !p.s || (stats && !p.part) || p.c_in < 1 || p.c_in > kStemPix || p.w > kStemMaxW ||
        p.ho != stem_out(p.h) || p.wo != stem_out(p.w))
        return hipErrorInvalidValue;
    const int64_t m = (int64_t)p.n * p.ho * p.wo;
    const double e = dtype == DT_BF16 ? 2.0 : 4.0;
    TraceScope tr(KC_CONV, KID_STEM_CONV, s, e * ((double)p.n * p.h * p.w * kStemPix + (double)m * kStemCout),
                  2.0 * m * kStemCout * kSK * kSK * p.c_in);
    if (dtype == DT_BF16) {
        const int64_t items = (int64_t)p.n * ((p.ho + kStemRows - 1) / kStemRows);
        const unsigned g = (unsigned)stem_groups(items);
        const size_t lds = stem_lds(p.wo, false);
        if (stats) hipLaunchKernelGGL(k_stem_conv<true>, dim3(g), dim3(kThreads), lds, s, p);
        else hipLaunchKernelGGL(k_stem_conv<false>, dim3(g), dim3(kThreads), lds, s, p);
    } else {
        const int64_t total = m * kStemCout;
        const unsigned g = (unsigned)(ceil_div(total, kThreads) < 8192 ? ceil_div(total, kThreads) : 8192);
        hipLaunchKernelGGL(k_stem_conv_f32, dim3(g), dim3(kThreads), 0, s, p);
    }
    return hipGetLastError();
}

int64_t stem_wgrad_splits(int dtype, int64_t items) { return dtype == DT_BF16 ? stem_groups(items) : 1; }

hipError_t launch_stem_wgrad(int dtype, const StemParams &p, int gsrc, hipStream_t s)
{
    if (!p.img || !p.g || !p.dwpart || p.c_in < 1 || p.c_in > kStemPix || p.w > kStemMaxW ||
        p.ho != stem_out(p.h) || p.wo != stem_out(p.w) ||
        (gsrc == GB_BNGRAD && (!p.gx || !p.g_gamma || !p.g_mean || !p.g_rstd || !p.g_dgamma || !p.g_dbeta)) ||
        (gsrc != GB_BNGRAD && gsrc != GB_DENSE))
        return hipErrorInvalidValue;
    const int64_t m = (int64_t)p.n * p.ho * p.wo;
    const double e = dtype == DT_BF16 ? 2.0 : 4.0;
    const double nw = (double)kSK * kSK * p.c_in * kStemCout;
    const double gbytes = e * (double)m * kStemCout * (gsrc == GB_BNGRAD ? 2.0 : 1.0);
    TraceScope tr(KC_WGRAD, KID_STEM_WGRAD, s, e * (double)p.n * p.h * p.w * kStemPix + gbytes + 4.0 * nw,
                  2.0 * m * nw);
    if (dtype == DT_BF16) {
        const int64_t items = (int64_t)p.n * ((p.ho + kStemRows - 1) / kStemRows);
        const unsigned g = (unsigned)stem_groups(items);
        const size_t lds = stem_lds(p.wo, true);
        if (gsrc == GB_BNGRAD) hipLaunchKernelGGL(k_stem_wgrad<GB_BNGRAD>, dim3(g), dim3(kThreads), lds, s, p);
        else hipLaunchKernelGGL(k_stem_wgrad<GB_DENSE>, dim3(g), dim3(kThreads), lds, s, p);
    } else {
        const unsigned g = (unsigned)ceil_div((int64_t)nw, kThreads);
        if (gsrc == GB_BNGRAD) hipLaunchKernelGGL(k_stem_wgrad_f32<GB_BNGRAD>, dim3(g), dim3(kThreads), 0, s, p);
        else hipLaunchKernelGGL(k_stem_wgrad_f32<GB_DENSE>, dim3(g), dim3(kThreads), 0, s, p);
    }
    return hipGetLastError();
}

int64_t maxpool_fwd_rows(int dtype, int64_t m_out, int c) { return stats_row_blocks(m_out, c, dtype); }

hipError_t launch_maxpool_fwd(int dtype, const MaxPoolParams &p, bool bn, bool stats, hipStream_t s)
{
    if (!p.x || !p.y || (bn && (!p.gamma || !p.beta || !p.mean || !p.rstd)) || (stats && !p.part) ||
        p.ho != (p.h - 1) / 2 + 1 || p.wo != (p.w - 1) / 2 + 1)
        return hipErrorInvalidValue;
    const int64_t m_out = (int64_t)p.n * p.ho * p.wo;
    const int64_t R = maxpool_fwd_rows(dtype, m_out, p.c);
    const int64_t rpb = ceil_div(m_out, R);
    const int cb = (int)ceil_div(p.c, stats_ch_per_block(dtype));
    dim3 grid((unsigned)ceil_div(m_out, rpb), (unsigned)cb);
    const double e = dtype == DT_BF16 ? 2.0 : 4.0;
    TraceScope tr(KC_SWEEP, KID_MAXPOOL, s, e * p.c * ((double)p.n * p.h * p.w + (double)m_out), 0.0);
    auto go = [&](auto kern) { hipLaunchKernelGGL(kern, grid, dim3(kThreads), 0, s, p, rpb); };
    if (dtype == DT_BF16) {
        if (bn) { if (stats) go(k_maxpool_fwd<bf16_t, true, true>); else go(k_maxpool_fwd<bf16_t, true, false>); }
        else { if (stats) go(k_maxpool_fwd<bf16_t, false, true>); else go(k_maxpool_fwd<bf16_t, false, false>); }
    } else {
        if (bn) { if (stats) go(k_maxpool_fwd<float, true, true>); else go(k_maxpool_fwd<float, true, false>); }
        else { if (stats) go(k_maxpool_fwd<float, false, true>); else go(k_maxpool_fwd<float, false, false>); }
    }
    return hipGetLastError();
}

int64_t maxpool_bwd_groups(int n, int h)
{
    const int64_t items = (int64_t)n * ((h + 1) / 2);
    return items < kMaxPoolBwdGroups ? (items < 1 ? 1 : items) : kMaxPoolBwdGroups;
}

hipError_t launch_maxpool_bwd(int dtype, const MaxPoolParams &p, bool bn, hipStream_t s)
{
    const int vec = dtype == DT_BF16 ? 8 : 4, cvec = p.c / vec;
    if (!p.x || !p.g || !p.y || (bn && (!p.gamma || !p.beta || !p.mean || !p.rstd || !p.part)) ||
        p.c > kMaxPoolMaxC || p.wo > kMaxPoolMaxWo || cvec < 1 || (kThreads % cvec) ||
        p.ho != (p.h - 1) / 2 + 1 || p.wo != (p.w - 1) / 2 + 1)
        return hipErrorInvalidValue;
    const unsigned g = (unsigned)maxpool_bwd_groups(p.n, p.h);
    const double e = dtype == DT_BF16 ? 2.0 : 4.0, m = (double)p.n * p.h * p.w;
    TraceScope tr(KC_SWEEP, KID_MAXPOOL, s, e * p.c * ((bn ? 2.0 : 1.0) * m + (double)p.n * p.ho * p.wo), 0.0);
    if (dtype == DT_BF16) {
        if (bn) hipLaunchKernelGGL((k_maxpool_bwd<bf16_t, true>), dim3(g), dim3(kThreads), 0, s, p);
        else hipLaunchKernelGGL((k_maxpool_bwd<bf16_t, false>), dim3(g), dim3(kThreads), 0, s, p);
    } else {
        if (bn) hipLaunchKernelGGL((k_maxpool_bwd<float, true>), dim3(g), dim3(kThreads), 0, s, p);
        else hipLaunchKernelGGL((k_maxpool_bwd<float, false>), dim3(g), dim3(kThreads), 0, s, p);
    }
    return hipGetLastError();
}

hipError_t launch_head_fwd(int dtype, const HeadParams &p, hipStream_t s)
{
    if (!p.x || !p.gamma || !p.beta || !p.mean || !p.rstd || !p.f || !p.wfc || !p.bfc || !p.labels || !p.logits ||
        !p.dlogits || !p.loss)
        return hipErrorInvalidValue;
    const int vec = dtype == DT_BF16 ? 8 : 4;
    const double e = dtype == DT_BF16 ? 2.0 : 4.0;
    TraceScope tr(KC_SMALL, KID_HEAD, s,
                  e * ((double)p.n * p.h * p.w * p.c + (double)p.c * p.classes) + 8.0 * p.n * p.classes,
                  2.0 * p.n * p.c * p.classes);
    const int nt = p.n * (p.c / vec);
    if (dtype == DT_BF16) hipLaunchKernelGGL(k_head_pool<bf16_t>, dim3((unsigned)ceil_div(nt, kThreads)), dim3(kThreads), 0, s, p);
    else hipLaunchKernelGGL(k_head_pool<float>, dim3((unsigned)ceil_div(nt, kThreads)), dim3(kThreads), 0, s, p);
    dim3 grid((unsigned)ceil_div(p.classes, kFcBN), (unsigned)ceil_div(p.n, 16));
    if (dtype == DT_BF16)
        hipLaunchKernelGGL(k_fc_gemm<bf16_t>, grid, dim3(kThreads), 0, s, p.n, p.classes, p.c, p.f, (int64_t)p.c,
                           (int64_t)1, (const bf16_t *)p.wfc, (int64_t)p.classes, (int64_t)1, p.bfc, p.logits);
    else
        hipLaunchKernelGGL(k_fc_gemm<float>, grid, dim3(kThreads), 0, s, p.n, p.classes, p.c, p.f, (int64_t)p.c,
                           (int64_t)1, (const float *)p.wfc, (int64_t)p.classes, (int64_t)1, p.bfc, p.logits);
    hipLaunchKernelGGL(k_softmax_ce, dim3((unsigned)p.n), dim3(kThreads), 0, s, p.n, p.classes, p.logits, p.labels,
                       p.dlogits, p.loss);
    hipLaunchKernelGGL(k_loss_mean, dim3(1), dim3(64), 0, s, p.n, p.loss);
    return hipGetLastError();
}

int64_t head_rows(int dtype, int64_t m, int c) { return stats_row_blocks(m, c, dtype); }

hipError_t launch_head_bwd_fc(int dtype, const HeadParams &p, hipStream_t s)
{
    if (!p.f || !p.wfc || !p.dlogits || !p.df || !p.dwfc || !p.dbfc) return hipErrorInvalidValue;
    TraceScope tr(KC_SMALL, KID_HEAD, s, 4.0 * ((double)p.n * p.classes + 2.0 * p.n * p.c + (double)p.c * p.classes),
                  4.0 * p.n * p.c * p.classes);
    // df = dlogits W^T: A = dlogits [n][K], B(k=j, col=c) = W[c][j]
    dim3 g1((unsigned)ceil_div(p.c, kFcBN), (unsigned)ceil_div(p.n, 16));
    if (dtype == DT_BF16)
        hipLaunchKernelGGL(k_fc_gemm<bf16_t>, g1, dim3(kThreads), 0, s, p.n, p.c, p.classes, p.dlogits,
                           (int64_t)p.classes, (int64_t)1, (const bf16_t *)p.wfc, (int64_t)1, (int64_t)p.classes,
                           (const float *)nullptr, p.df);
    else
        hipLaunchKernelGGL(k_fc_gemm<float>, g1, dim3(kThreads), 0, s, p.n, p.c, p.classes, p.dlogits,
                           (int64_t)p.classes, (int64_t)1, (const float *)p.wfc, (int64_t)1, (int64_t)p.classes,
                           (const float *)nullptr, p.df);
    // dW = f^T dlogits: A(i=c, k=n) = f[n][c], B(k=n, j) = dlogits[n][j]
    dim3 g2((unsigned)ceil_div(p.classes, kFcBN), (unsigned)ceil_div(p.c, 16));
    hipLaunchKernelGGL(k_fc_gemm<float>, g2, dim3(kThreads), 0, s, p.c, p.classes, p.n, p.f, (int64_t)1,
                       (int64_t)p.c, p.dlogits, (int64_t)p.classes, (int64_t)1, (const float *)nullptr, p.dwfc);
    hipLaunchKernelGGL(k_colsum, dim3((unsigned)ceil_div(p.classes, kThreads)), dim3(kThreads), 0, s, p.n, p.classes,
                       p.dlogits, p.dbfc);
    return hipGetLastError();
}

hipError_t launch_head_bn_bwd(int dtype, const HeadParams &p, int mode, hipStream_t s)
{
    if (!p.x || !p.gamma || !p.beta || !p.mean || !p.rstd || !p.df || (mode != HB_SUMS && !p.gx) ||
        (mode != HB_DX && !p.part) || (mode == HB_DX && (!p.dgamma || !p.dbeta)))
        return hipErrorInvalidValue;
    const int64_t m = (int64_t)p.n * p.h * p.w;
    const int64_t R = head_rows(dtype, m, p.c);
    const int64_t rpb = ceil_div(m, R);
    const int cb = (int)ceil_div(p.c, stats_ch_per_block(dtype));
    dim3 grid((unsigned)ceil_div(m, rpb), (unsigned)cb);
    const double e = dtype == DT_BF16 ? 2.0 : 4.0;
    TraceScope tr(KC_SMALL, KID_HEAD, s, e * (double)m * p.c * (mode == HB_SUMS ? 1.0 : 2.0) + 4.0 * p.n * p.c, 0.0);
    auto go = [&](auto kern) { hipLaunchKernelGGL(kern, grid, dim3(kThreads), 0, s, p, rpb); };
    if (dtype == DT_BF16) {
        if (mode == HB_SPLIT) go(k_head_bn_bwd<bf16_t, HB_SPLIT>);
        else if (mode == HB_SUMS) go(k_head_bn_bwd<bf16_t, HB_SUMS>);
        else go(k_head_bn_bwd<bf16_t, HB_DX>);
    } else {
        if (mode == HB_SPLIT) go(k_head_bn_bwd<float, HB_SPLIT>);
        else if (mode == HB_SUMS) go(k_head_bn_bwd<float, HB_SUMS>);
        else go(k_head_bn_bwd<float, HB_DX>);
    }
    return hipGetLastError();
}

}  // namespace bnr
