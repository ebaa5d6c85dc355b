// Device-side helpers for the gfx950 kernels: element types, MFMA operand
// traits, wavefront scans.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace m3 {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;      // CDNA wavefront width
constexpr int kBlock = 256;    // threads per workgroup (4 waves)

__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(bf16 v) { return static_cast<float>(v); }

template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float v) {
    return static_cast<bf16>(v);   // round to nearest even
}

// MFMA 16x16 output tiles.  Operand fragment of lane l (g = l / 16):
//   A: row l % 16, K-elements KPL*g .. KPL*g + KPL-1 of the K-step
//   B: column l % 16, same K-elements
//   C/D: column l % 16, rows 4*g .. 4*g + 3
template <typename T> struct Mma;

template <> struct Mma<bf16> {
    static constexpr int K = 32;     // v_mfma_f32_16x16x32_bf16
    static constexpr int KPL = 8;
    typedef bf16x8 frag;
    __device__ static __forceinline__ f32x4 mma(frag a, frag b, f32x4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
    __device__ static __forceinline__ frag load(const bf16 *p) {
        return *reinterpret_cast<const bf16x8 *>(p);
    }
};

template <> struct Mma<float> {
    static constexpr int K = 4;      // v_mfma_f32_16x16x4_f32
    static constexpr int KPL = 1;
    typedef float frag;
    __device__ static __forceinline__ f32x4 mma(frag a, frag b, f32x4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
    }
    __device__ static __forceinline__ frag load(const float *p) { return *p; }
};

// Scalar type of the prologue (chunk-local prefix sums of log-decays and
// angles, their exponentials and rotations).  The fp32 build keeps these in
// fp64 so that differences of prefix sums stay exact to fp32 rounding.
template <typename T> struct AccOf { typedef float type; };
template <> struct AccOf<float> { typedef double type; };

__device__ __forceinline__ void sincos_acc(float x, float *s, float *c) { sincosf(x, s, c); }
__device__ __forceinline__ void sincos_acc(double x, double *s, double *c) { sincos(x, s, c); }
__device__ __forceinline__ float exp_acc(float x) { return expf(x); }
__device__ __forceinline__ double exp_acc(double x) { return exp(x); }

// Hardware transcendentals for the bf16 path (v_sin/v_cos/v_exp after an
// explicit reduction of the angle to [-pi, pi]; errors ~1e-6 relative, far
// below bf16 rounding), and accurate fp64 for the fp32 path.
__device__ __forceinline__ float reduce_angle(float x) {
    return x - 6.28318530717958647692f * rintf(x * 0.15915494309189533577f);
}
__device__ __forceinline__ void sincos_fast(float x, float *s, float *c) {
    __sincosf(reduce_angle(x), s, c);
}
__device__ __forceinline__ void sincos_fast(double x, double *s, double *c) { sincos(x, s, c); }
__device__ __forceinline__ float exp_fast(float x) { return __expf(x); }
// 2^x on the hardware exp unit (v_exp_f32)
__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ double exp_fast(double x) { return exp(x); }

// SiLU(u) = u / (1 + e^{-u}), the output gate's activation (App. "MIMO for
// Mamba-3": Y' = Y o SiLU(Z)).  Hardware exp and reciprocal (~1e-7 relative);
// e^{-u} overflowing to +inf for very negative u gives the limit -0.
__device__ __forceinline__ float silu(float u) {
    return u * __builtin_amdgcn_rcpf(1.f + __expf(-u));
}

// Inclusive prefix sum across the 64 lanes of a wavefront.
template <typename A>
__device__ __forceinline__ A wave_incl_scan(A v, int lane) {
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        A n = __shfl_up(v, o, kWave);
        if (lane >= o) v += n;
    }
    return v;
}

}  // namespace m3
