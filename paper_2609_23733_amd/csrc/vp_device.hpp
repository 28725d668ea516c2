// Device helpers shared by the gfx950 kernels of the routed global-attention
// layer: vector types, bf16 conversion, MFMA wrappers, wave reductions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace vp {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef __bf16 bf16x4 __attribute__((__vector_size__(4 * sizeof(__bf16))));
typedef __bf16 bf16x2 __attribute__((__vector_size__(2 * sizeof(__bf16))));
typedef _Float16 f16;
typedef _Float16 f16x8 __attribute__((__vector_size__(8 * sizeof(_Float16))));
typedef _Float16 f16x2 __attribute__((__vector_size__(2 * sizeof(_Float16))));
typedef float f32x16 __attribute__((__vector_size__(16 * sizeof(float))));
typedef float f32x4 __attribute__((__vector_size__(4 * sizeof(float))));
typedef float f32x2 __attribute__((__vector_size__(2 * sizeof(float))));
typedef uint32_t u32x4 __attribute__((__vector_size__(4 * sizeof(uint32_t))));

constexpr int kD = 64;        // head dimension
constexpr int kL = 64;        // router / surrogate hidden size
constexpr int kMaxHeads = 16;
constexpr int kBucketsLen = 3 + kMaxHeads + 1;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

enum { DT_F32 = 0, DT_BF16 = 1 };
enum { MODE_MEAN = 0, MODE_SURR = 1, MODE_FULL = 2 };

__device__ __forceinline__ float exp2f_fast(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float rcp_fast(float x) { return __builtin_amdgcn_rcpf(x); }

__device__ __forceinline__ float bf16_to_f32(bf16 x) { return (float)x; }

// GELU(x) = x Phi(x) = (x / 2) (1 + erf(x / sqrt 2)), with erf from the rational
// approximation 7.1.26 of Abramowitz and Stegun (Handbook of Mathematical
// Functions): erf(z) = 1 - (a1 t + ... + a5 t^5) e^{-z^2}, t = 1 / (1 + p z),
// z >= 0, absolute error <= 1.5e-7, odd extension for z < 0.  For fp32
// outputs.
__device__ __forceinline__ float gelu_erf(float x) {
    const float z = fabsf(x) * 0.70710678118654752f;
    const float t = rcp_fast(fmaf(0.3275911f, z, 1.f));
    float q = fmaf(1.061405429f, t, -1.453152027f);
    q = fmaf(q, t, 1.421413741f);
    q = fmaf(q, t, -0.284496736f);
    q = fmaf(q, t, 0.254829592f);
    q *= t;
    const float e = exp2f_fast(-z * z * kLog2e);
    const float erfz = fmaf(-q, e, 1.f);                       // erf(|x| / sqrt 2)
    const float phi2 = 1.f + (x < 0.f ? -erfz : erfz);         // 1 + erf(x / sqrt 2)
    return 0.5f * x * phi2;
}

// GELU for bf16 outputs: Phi(x) ~ sigmoid(g(x)) with g odd,
// g(x) = x (a1 + a3 x^2 + a5 x^4) for |x| <= 6 and g(+-6) beyond
// (Phi(6) = 1 - 1e-9).  The coefficients minimise
// the largest GELU error over [-7, 7]; evaluated in fp32 the error is at most
// 2.6e-5 anywhere, below the bf16 rounding of the activations the bf16
// kernels store.  Seven vector instructions and two transcendental ones
// (exp2, reciprocal), against fifteen and two for gelu_erf.
constexpr float kGeluA1 = 1.59501577f, kGeluA3 = 7.40112920e-02f, kGeluA5 = -7.03033577e-04f;
__device__ __forceinline__ float gelu(float x) {
    const float xc = __builtin_amdgcn_fmed3f(x, -6.f, 6.f);
    const float x2 = xc * xc;
    const float g = xc * fmaf(x2, fmaf(x2, kGeluA5 * kLog2e, kGeluA3 * kLog2e), kGeluA1 * kLog2e);
    return x * rcp_fast(1.f + exp2f_fast(-g));   // x sigmoid(g), g in log2 units
}

// 32x32x16 bf16 MFMA, fp32 accumulate (gfx950).  Operand layout, lane l:
//   A[m][k]: m = l % 32, k = 8 * (l / 32) + j  (j = 0..7 of the bf16x8)
//   B[k][n]: n = l % 32, k = 8 * (l / 32) + j
//   D[m][n]: n = l % 32, m = 8 * (r / 4) + 4 * (l / 32) + (r % 4), r = 0..15
__device__ __forceinline__ f32x16 mfma_bf16(bf16x8 a, bf16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// 32x32x16 fp16 MFMA, fp32 accumulate; same operand layout as the bf16 one.
__device__ __forceinline__ f32x16 mfma_f16(f16x8 a, f16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

// 32x32x2 fp32 MFMA: A[m][k]: m = l % 32, k = l / 32; B[k][n]: n = l % 32,
// k = l / 32; D as above.
__device__ __forceinline__ f32x16 mfma_f32(float a, float b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

// Row (within a 32-row MFMA block) that holds key/feature `i` when the
// operand rows are stored with bits 2 and 3 of the index swapped.  With that
// order, output register r of lane-half hh of a 32x32 MFMA holds index
// 16 * (r / 8) + 8 * hh + (r % 8): eight consecutive indices per half, the
// layout the next MFMA's K operand needs.
__device__ __forceinline__ int swap23(int i) {
    return (i & ~12) | ((i & 4) << 1) | ((i & 8) >> 1);
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o);
    return x;
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
    return x;
}

__device__ __forceinline__ bf16x8 load_bf16x8(const bf16* p) {
    return *reinterpret_cast<const bf16x8*>(p);
}

__device__ __forceinline__ bf16x8 zero_bf16x8() {
    u32x4 z = {0u, 0u, 0u, 0u};
    return __builtin_bit_cast(bf16x8, z);
}

__device__ __forceinline__ f32x16 zero_f32x16() {
    f32x16 z;
#pragma unroll
    for (int i = 0; i < 16; ++i) z[i] = 0.f;
    return z;
}

// Pack eight fp32 values into bf16x8 with round-to-nearest-even.
__device__ __forceinline__ bf16x8 pack_bf16x8(float a0, float a1, float a2, float a3, float a4,
                                              float a5, float a6, float a7) {
    bf16x8 r;
    r[0] = (bf16)a0; r[1] = (bf16)a1; r[2] = (bf16)a2; r[3] = (bf16)a3;
    r[4] = (bf16)a4; r[5] = (bf16)a5; r[6] = (bf16)a6; r[7] = (bf16)a7;
    return r;
}

// Remap a linear work index so that consecutive work items land on the same
// XCD.  The dispatcher assigns workgroup i to XCD i % 8; item k of XCD x then
// receives work index x * q + min(x, r) + k over `active` items (q = active / 8,
// r = active % 8), a bijection of [0, active).
__device__ __forceinline__ int xcd_remap(int i, int active) {
    int q = active >> 3, r = active & 7;
    int x = i & 7, k = i >> 3;
    return x * q + (x < r ? x : r) + k;
}

}  // namespace vp
