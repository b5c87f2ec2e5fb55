// Device-side building blocks shared by the kve kernels (gfx950 / CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kve {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.44269504088896340736f;
constexpr int kWave = 64;

__device__ __forceinline__ u32x4 ld16(const void* p) {
    return *reinterpret_cast<const u32x4*>(p);
}
__device__ __forceinline__ void st16(void* p, u32x4 v) {
    *reinterpret_cast<u32x4*>(p) = v;
}
__device__ __forceinline__ u32x4 zero16() {
    u32x4 z = {0u, 0u, 0u, 0u};
    return z;
}

// exp2 on the transcendental unit (v_exp_f32): exact 0 for -inf.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// One 32x32 output block of a matrix-core product, accumulated over k.
//
// Operand layout of a 32x32 block on a 64-lane wave (shared by both types):
//   A (rows)  lane l supplies row  l%32,  k-values kbase(s, l) .. + KPL
//   B (cols)  lane l supplies col  l%32,  the same k-values
//   C         lane l holds col l%32 and rows 8*(i/4) + 4*(l/32) + (i%4), i < 16
// kbase(s, l) = s*KSTEP + (l/32)*KPL: step s covers KSTEP consecutive k values,
// the lower half of the wave the first KPL of them.
template <typename T> struct Mma;

template <> struct Mma<__bf16> {
    static constexpr int KSTEP = 16;
    static constexpr int KPL = 8;
    typedef bf16x8 frag;
    __device__ __forceinline__ static frag load(const void* row, int k) {
        return *reinterpret_cast<const bf16x8*>(reinterpret_cast<const __bf16*>(row) + k);
    }
    __device__ __forceinline__ static frag zero() {
        frag z;
        for (int e = 0; e < 8; ++e) z[e] = (__bf16)0.0f;
        return z;
    }
    __device__ __forceinline__ static f32x16 mma(frag a, frag b, f32x16 c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
    }
};

template <> struct Mma<float> {
    static constexpr int KSTEP = 2;
    static constexpr int KPL = 1;
    typedef float frag;
    __device__ __forceinline__ static frag load(const void* row, int k) {
        return reinterpret_cast<const float*>(row)[k];
    }
    __device__ __forceinline__ static frag zero() { return 0.0f; }
    __device__ __forceinline__ static f32x16 mma(frag a, frag b, f32x16 c) {
        return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
    }
};

// 16 bytes of a key or value row as CW floats.
template <typename T>
struct VPiece;

template <>
struct VPiece<__bf16> {
    static constexpr int CW = 8;
    __device__ __forceinline__ static void to_f(u32x4 v, float (&f)[CW]) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            f[2 * e] = __uint_as_float(v[e] << 16);
            f[2 * e + 1] = __uint_as_float(v[e] & 0xffff0000u);
        }
    }
};

template <>
struct VPiece<float> {
    static constexpr int CW = 4;
    __device__ __forceinline__ static void to_f(u32x4 v, float (&f)[CW]) {
#pragma unroll
        for (int e = 0; e < 4; ++e) f[e] = __uint_as_float(v[e]);
    }
};

// x[l] + x[l ^ 32] in every lane l: the two halves of the wave swapped with
// v_permlane32_swap (a vector-unit instruction of gfx950) and added; the sum of
// the swap's two results is the same whichever half each result holds.
__device__ __forceinline__ float half_wave_sum(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Row of output register i held by lane l in a 32x32 block (see Mma).
__device__ __forceinline__ int c_row(int i, int lane) {
    return 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
}

// Merge two (max, sum-of-exp2) pairs of the same row.  -inf max means empty.
__device__ __forceinline__ void lse2_merge(float& m, float& l, float mo, float lo) {
    const float mn = fmaxf(m, mo);
    if (mn == -INFINITY) {
        m = mn;
        l = 0.0f;
        return;
    }
    l = l * fast_exp2(m - mn) + lo * fast_exp2(mo - mn);
    m = mn;
}

// Order-preserving map of a float32 score to an unsigned key (larger score,
// larger key).  -0.0 maps like +0.0; every NaN maps to 0, below -inf.
__device__ __forceinline__ uint32_t score_key(float f) {
    uint32_t b = __float_as_uint(f);
    if ((b & 0x7fffffffu) > 0x7f800000u) return 0u;
    if (b == 0x80000000u) b = 0u;
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

}  // namespace kve
