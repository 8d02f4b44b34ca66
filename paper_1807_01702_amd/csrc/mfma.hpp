// mfma.hpp -- the two gfx950 matrix-core forms the CONV kernels use.
//
// v_mfma_f32_16x16x32_bf16: lane l holds A[l%16][8*(l/16) + e] and
// B[8*(l/16) + e][l%16] for e = 0..7 and accumulates C[4*(l/16) + i][l%16],
// i = 0..3.  v_mfma_f32_16x16x4_f32: same with one k per lane (k = l/16).
// (Lane layouts checked on the device with an in-bounds probe.)
#pragma once
#include "common.hpp"

namespace bnr {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <typename T> struct Mfma;

template <> struct Mfma<bf16_t> {
    static constexpr int KPL = 8;      // k values per lane
    static constexpr int KSTEP = 32;   // k per instruction
    typedef bf16x8 frag;
    __device__ static __forceinline__ frag load(const bf16_t *p) {
        return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(p));
    }
    __device__ static __forceinline__ frag zero() { u32x4 z = {0u, 0u, 0u, 0u}; return __builtin_bit_cast(bf16x8, z); }
    __device__ static __forceinline__ frag from_words(const uint32_t *w) {
        u32x4 v = {w[0], w[1], w[2], w[3]};
        return __builtin_bit_cast(bf16x8, v);
    }
    __device__ static __forceinline__ void mma(f32x4 &c, frag a, frag b) {
        c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
    // c = a b (a zero accumulator as the inline constant: no register clears)
    __device__ static __forceinline__ void mma0(f32x4 &c, frag a, frag b) {
        const f32x4 z = {0.f, 0.f, 0.f, 0.f};
        c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, z, 0, 0, 0);
    }
};

template <> struct Mfma<float> {
    static constexpr int KPL = 1;
    static constexpr int KSTEP = 4;
    typedef float frag;
    __device__ static __forceinline__ frag load(const float *p) { return *p; }
    __device__ static __forceinline__ frag zero() { return 0.f; }
    __device__ static __forceinline__ void mma(f32x4 &c, frag a, frag b) {
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
    }
};

// bf16 matrix-core fragment of 8 consecutive rows of one column from a
// row-major LDS tile with the given row pitch (elements), by two transposing
// 8-byte reads (ds_read_b64_tr_b16): within a group of 16 lanes, lane j
// reads the 4 columns 4 (j % 4) .. +3 of row j / 4 and lane i receives
// column i of rows 0..3; p is this lane's address of row j / 4 (+ 8 g for
// lane group g), column 4 (j % 4).
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

__device__ __forceinline__ bf16x8 tr_frag(const bf16_t *p, int pitch)
{
    const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(p));
    const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(p + 4 * pitch));
    typedef short s16x8 __attribute__((ext_vector_type(8)));
    const s16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    return __builtin_bit_cast(bf16x8, v);
}

// round an fp32 value to the storage type T (bf16: RNE)
template <typename T> __device__ __forceinline__ T to_store(float f);
template <> __device__ __forceinline__ float to_store<float>(float f) { return f; }
template <> __device__ __forceinline__ bf16_t to_store<bf16_t>(float f) { return f2bf(f); }

}  // namespace bnr
