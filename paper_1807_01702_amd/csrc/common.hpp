// common.hpp -- device helpers shared by the libbnr kernels (gfx950 only).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bnr {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint16_t bf16_t;   // bf16 storage word

struct alignas(16) vec16 { uint32_t u[4]; };

constexpr int kThreads = 256;   // every kernel runs 256-thread workgroups (4 waves of 64)

__device__ __forceinline__ float bf2f(bf16_t h) { return __uint_as_float((uint32_t)h << 16); }
// float -> bf16, round to nearest even (v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ bf16_t f2bf(float f) {
    __bf16 b = (__bf16)f;
    bf16_t u;
    __builtin_memcpy(&u, &b, 2);
    return u;
}
// two floats -> packed bf16 pair (one v_cvt_pk_bf16_f32)
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack2bf(float lo, float hi) {
    const f32x2_t f = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2_t));
}

// Element traits: VEC = elements per 16-byte vector; storage <-> float.
template <typename T> struct Elem;
template <> struct Elem<float> {
    static constexpr int VEC = 4;
    __device__ static __forceinline__ void unpack(const vec16 &v, float *f) {
        for (int i = 0; i < 4; i++) f[i] = __uint_as_float(v.u[i]);
    }
    __device__ static __forceinline__ vec16 pack(const float *f) {
        vec16 v;
        for (int i = 0; i < 4; i++) v.u[i] = __float_as_uint(f[i]);
        return v;
    }
    __device__ static __forceinline__ float round(float f) { return f; }
    __device__ static __forceinline__ float load1(const float *p) { return *p; }
    __device__ static __forceinline__ float from(float s) { return s; }
};
template <> struct Elem<bf16_t> {
    static constexpr int VEC = 8;
    __device__ static __forceinline__ void unpack(const vec16 &v, float *f) {
        for (int i = 0; i < 4; i++) {
            f[2 * i] = __uint_as_float(v.u[i] << 16);
            f[2 * i + 1] = __uint_as_float(v.u[i] & 0xffff0000u);
        }
    }
    __device__ static __forceinline__ vec16 pack(const float *f) {
        vec16 v;
        for (int i = 0; i < 4; i++) v.u[i] = pack2bf(f[2 * i], f[2 * i + 1]);
        return v;
    }
    __device__ static __forceinline__ float round(float f) { return bf2f(f2bf(f)); }
};

__device__ __forceinline__ vec16 ldg16(const void *p) { return *reinterpret_cast<const vec16 *>(p); }
// Streaming load of data read once (non-temporal: no reuse expected in the caches).
__device__ __forceinline__ vec16 ldg16_stream(const void *p) {
    const vec16 *s = reinterpret_cast<const vec16 *>(p);
    vec16 v;
    for (int k = 0; k < 4; k++) v.u[k] = __builtin_nontemporal_load(&s->u[k]);
    return v;
}
__device__ __forceinline__ void stg16(void *p, const vec16 &v) { *reinterpret_cast<vec16 *>(p) = v; }
__device__ __forceinline__ vec16 zero16() { vec16 v; v.u[0] = v.u[1] = v.u[2] = v.u[3] = 0; return v; }

// Raw buffer view of [base, base + bytes) (bytes < 2^31).  A load at an
// offset outside the range returns zeros in hardware, so operand loads need
// neither a branch nor a zero-initialised destination (which would force the
// compiler to wait for older memory operations before issuing them).
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
constexpr uint32_t kBufOff = 0x80000000u;       // an offset that is always out of range
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_view(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ vec16 bld16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    const u32x4_t t = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
    vec16 v;
    v.u[0] = t.x; v.u[1] = t.y; v.u[2] = t.z; v.u[3] = t.w;
    return v;
}
// Store through a raw buffer view: an out-of-range offset (kBufOff) drops the
// store, so a masked row needs no branch.
__device__ __forceinline__ void bst16(__amdgpu_buffer_rsrc_t r, uint32_t off, const vec16 &v) {
    const u32x4_t t = {v.u[0], v.u[1], v.u[2], v.u[3]};
    __builtin_amdgcn_raw_buffer_store_b128(t, r, off, 0, 0);
}

// Column sums of two float arrays in LDS, a = red[0 .. rows)[ld] and
// b = red[rows .. 2 rows)[ld], columns 0 .. ncol-1, by all nthr threads of the
// workgroup: each thread sums a strided slice of one column's rows, then
// threads 0 .. 2 ncol-1 add the slices in order (a fixed order: the result
// is deterministic).  Writes outa[c], outb[c] for c < nvalid.  Starts and
// ends with a barrier; overwrites the first nthr floats of red.
__device__ __forceinline__ void lds_colsum2(float *red, int rows, int ld, int ncol, int nthr, int tid,
                                            float *outa, float *outb, int nvalid)
{
    const int lanes = 2 * ncol;
    int S = nthr / lanes;
    S = S < 1 ? 1 : (S > rows ? rows : S);
    const int lane = tid % lanes, slice = tid / lanes;
    float acc = 0.f;
    __syncthreads();
    if (slice < S) {
        const float *col = red + (lane < ncol ? lane : rows * ld + lane - ncol);
        for (int j = slice; j < rows; j += S) acc += col[j * ld];
    }
    __syncthreads();
    if (slice < S) red[slice * lanes + lane] = acc;
    __syncthreads();
    if (tid < lanes) {
        float t = 0.f;
        for (int q = 0; q < S; q++) t += red[q * lanes + tid];
        const int c = tid < ncol ? tid : tid - ncol;
        if (c < nvalid) (tid < ncol ? outa : outb)[c] = t;
    }
}

// sub-BN2 (normalise, scale, shift) as one fused multiply-add per element:
// y = x c0 + c1 with c0 = gamma rstd and c1 = beta - mean c0.  Every kernel
// that applies it before a ReLU (CONV prologues, the weight gradient's
// recompute, max pooling, the head) and every BN-backward epilogue that
// rebuilds the ReLU mask [y > 0] from x goes through these two helpers, so
// the forward output, the mask of dx and the recomputed dW operand take the
// same decision at every pixel, bit for bit.
__device__ __forceinline__ void bn_coef(float gamma, float beta, float mean, float rstd, float &c0, float &c1) {
    c0 = gamma * rstd;
    c1 = __builtin_fmaf(-mean, c0, beta);
}
__device__ __forceinline__ float bn_lin(float x, float c0, float c1) { return __builtin_fmaf(x, c0, c1); }

// Normalisation centre of a BN input held in float32.  A consumer may be given
// a centre K (the float32 mean) and the mean relative to it (mean - K: the low
// part of the float64 mean), and then normalises the centred value x - K:
//   y = (x - K) c0 + (beta - (mean - K) c0),  xhat = ((x - K) - (mean - K)) rstd,
// the deferred gradient d = A dy + B (x - K) + C with deferred_coef given
// mean - K.  Evaluated on x itself with the float32 mean, c1 = beta - mean c0
// and the product x c0 would carry |mean| 2^-24 of absolute error, more than
// the normalised value can afford once |mean| / std reaches 10^3; x - K is
// exact there (Sterbenz: operands within a factor of two).  bf16 storage
// already carries |x| 2^-9, so its consumers take K = 0: a compile-time zero,
// and x - 0 = x exactly (also for -0), so the subtraction folds away.
template <typename T>
__device__ __forceinline__ float bn_centre(const float *ctr, int c) {
    if constexpr (sizeof(T) == 4) return ctr ? ctr[c] : 0.f;
    else return 0.f;
}

// Deferred input gradient of a BN-fed tensor, formed on load as
//   d = A dy + B x + C  per channel (dy the loaded gradient, x the BN input).
// One BN (split = 0):  d = gamma rstd (dy - dbeta/m - xhat dgamma/m), i.e.
//   A = gamma rstd, B = -A rstd dgamma/m, C = A (rstd dgamma/m mean - dbeta/m).
// Several BNs reading the same channels with the same statistics (the
// consumers of a concatenated feature map, split = 1): the gradient buffer
// holds D = sum_l gamma_l rstd dy_l and the per-channel sums
// alpha = -sum_l gamma_l rstd dbeta_l/m, betap = -sum_l gamma_l rstd dgamma_l/m,
// so d = D + alpha + betap xhat: A = 1, B = betap rstd, C = alpha - B mean.
// The same from the channel's values: split = 1 takes (alpha, betap) in the
// places of (gamma, dgamma) and ignores dbeta.
__device__ __forceinline__ void deferred_coef_of(int split, float inv_m, float gamma, float mean, float rstd,
                                                 float dgamma, float dbeta, float &A, float &B, float &C)
{
    if (split) {
        A = 1.f;
        B = dgamma * rstd;
        C = gamma - B * mean;
    } else {
        const float k = gamma * rstd, b = dgamma * inv_m * rstd;
        A = k;
        B = -k * b;
        C = k * (b * mean - dbeta * inv_m);
    }
}
__device__ __forceinline__ void deferred_coef(int split, int c, float inv_m, const float *gamma, const float *mean,
                                              const float *rstd, const float *dgamma, const float *dbeta,
                                              const float *alpha, const float *betap, float &A, float &B, float &C)
{
    if (split) deferred_coef_of(1, inv_m, alpha[c], mean[c], rstd[c], betap[c], 0.f, A, B, C);
    else deferred_coef_of(0, inv_m, gamma[c], mean[c], rstd[c], dgamma[c], dbeta[c], A, B, C);
}

// Eight consecutive floats from a 32-byte aligned LDS address (two 16-byte reads).
__device__ __forceinline__ void lds_f8(const float *p, float *f) {
    const float4 a = reinterpret_cast<const float4 *>(p)[0], b = reinterpret_cast<const float4 *>(p)[1];
    f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w; f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
}

// Wave-level sum over the 64 lanes of a wave (all lanes get the result).
__device__ __forceinline__ float wave_sum(float v) {
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// Logical workgroup index for XCD-aware scheduling.  The dispatcher hands
// consecutive workgroup ids round-robin to the 8 XCDs (each with its own L2);
// this bijective remap gives every XCD a contiguous range of logical ids, so
// logically neighbouring tiles (halo rows, operands re-read by several output
// tiles) land on the same XCD and share its L2.
__device__ __forceinline__ int xcd_remap(int bid, int nblocks) {
    const int X = 8;
    const int q = nblocks / X, r = nblocks % X;
    const int x = bid % X, k = bid / X;
    return (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + k;
}

}  // namespace bnr
