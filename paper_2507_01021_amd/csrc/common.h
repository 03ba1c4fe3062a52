// Shared device helpers for the gfx950 kernels: bf16 storage type,
// conversions, vector types, wavefront reductions, error checks.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <stdexcept>
#include <string>

namespace wmi {

// bf16 as raw bits; arithmetic always happens in fp32.
struct bf16 {
    uint16_t x;
};

__host__ __device__ inline float bf2f(bf16 v) {
    union { uint32_t u; float f; } c;
    c.u = (uint32_t)v.x << 16;
    return c.f;
}

// fp32 -> bf16, round to nearest even (finite inputs; NaN stays NaN).
__host__ __device__ inline bf16 f2bf(float f) {
    union { uint32_t u; float f; } c;
    c.f = f;
    uint32_t u = c.u;
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x7fffffu)) {
        bf16 r; r.x = (uint16_t)((u >> 16) | 0x40); return r;
    }
    u += 0x7fffu + ((u >> 16) & 1u);
    bf16 r; r.x = (uint16_t)(u >> 16);
    return r;
}

// fp32 -> bf16 on the device with the hardware conversion (round to nearest
// even, same result as f2bf): two values packed into one 32-bit word.
__device__ inline uint32_t pack_bf16x2(float a, float b) {
    typedef float f32x2 __attribute__((ext_vector_type(2)));
    typedef __bf16 hbf16x2 __attribute__((ext_vector_type(2)));
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2{a, b}), hbf16x2));
}
__device__ inline bf16 f2bf_dev(float f) {
    bf16 r;
    r.x = __builtin_bit_cast(uint16_t, (__bf16)f);
    return r;
}

// Storage-type traits: load as fp32, store from fp32.
template <class T> struct St;
template <> struct St<float> {
    __device__ static inline float ld(const float* p) { return *p; }
    __device__ static inline void st(float* p, float v) { *p = v; }
};
template <> struct St<bf16> {
    __device__ static inline float ld(const bf16* p) { return bf2f(*p); }
    __device__ static inline void st(bf16* p, float v) { *p = f2bf_dev(v); }
};

template <class T> __device__ inline float ldf(const T* p) { return St<T>::ld(p); }
template <class T> __device__ inline void stf(T* p, float v) { St<T>::st(p, v); }

// Fragment-major layout of a matrix with K columns (K % 32 == 0), used for
// the bf16 decoder's projection weights and for the activations they
// multiply: the 16-row x 32-column block (row tile r / 16, k-step k / 32)
// is 1 KiB contiguous and holds, at byte 16 * l, what lane l of a 16x16x32
// MFMA operand needs (row l % 16, columns 8 * (l / 16) .. + 7). One
// operand fragment is therefore one fully contiguous 1 KiB load. Row tiles
// are stored one after another, each with all K / 32 k-steps.
__host__ __device__ inline long long frag_off(long long r, int k, int K) {
    return (((r >> 4) * (K >> 5) + (k >> 5)) * 64 + ((k >> 3) & 3) * 16 + (r & 15)) * 8 + (k & 7);
}
// Decoder matrices: fragment-major when stored as bf16, row-major as fp32.
template <class T>
__host__ __device__ inline long long dec_off(long long r, int k, int K) {
    if constexpr (sizeof(T) == 2) return frag_off(r, k, K);
    else return r * K + k;
}

// Native vectors (plain loads/stores; HIP's uint4 struct copies as memcpy).
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

// Four consecutive elements, stored with one 8-byte (bf16) or 16-byte (fp32) access.
__device__ inline void st4(float* p, float a, float b, float c, float d) {
    *reinterpret_cast<float4*>(p) = make_float4(a, b, c, d);
}
__device__ inline void st4(bf16* p, float a, float b, float c, float d) {
    const uint32_t lo = pack_bf16x2(a, b), hi = pack_bf16x2(c, d);
    *reinterpret_cast<u32x2*>(p) = u32x2{lo, hi};
}
__device__ inline float4 ld4(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ inline float4 ld4(const bf16* p) {
    const u32x2 u = *reinterpret_cast<const u32x2*>(p);
    union { uint32_t u; float f; } a, b, c, d;
    a.u = u.x << 16; b.u = u.x & 0xffff0000u; c.u = u.y << 16; d.u = u.y & 0xffff0000u;
    return make_float4(a.f, b.f, c.f, d.f);
}

// erf by Abramowitz & Stegun, Handbook of Mathematical Functions, formula
// 7.1.26 (absolute error below 1.5e-7): for z >= 0,
// erf(z) = 1 - t (a1 + t (a2 + t (a3 + t (a4 + t a5)))) exp(-z^2), t = 1 / (1 + p z).
__device__ inline float erf_as(float z) {
    const float az = fabsf(z);
    const float t = __builtin_amdgcn_rcpf(1.0f + 0.3275911f * az);
    const float poly = t * (0.254829592f + t * (-0.284496736f + t * (1.421413741f + t * (-1.453152027f + t * 1.061405429f))));
    const float r = 1.0f - poly * __expf(-az * az);
    return copysignf(r, z);
}
// GELU, erf form: x * Phi(x) = 0.5 x (1 + erf(x / sqrt 2)).
__device__ inline float gelu_erf(float x) { return 0.5f * x * (1.0f + erf_as(x * 0.70710678118654752f)); }

// 2^x for softmax weights (x at most a few units above 0, or -inf for
// masked terms): the hardware exponential alone, without the library
// wrapper's rescaling of results below the normal range (such weights are
// negligible next to the row maximum's weight of at least 1).
__device__ inline float exp2_softmax(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ inline float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}
__device__ inline float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
    return v;
}

// Order-preserving map of fp32 to uint32: a < b as floats (not NaN) iff
// f2ord(a) < f2ord(b) as integers. Host and device (the greedy-choice keys
// are checked on the host too).
__host__ __device__ inline uint32_t f2ord(float f) {
    const uint32_t u = __builtin_bit_cast(uint32_t, f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__host__ __device__ inline float ord2f(uint32_t o) {
    const uint32_t u = (o & 0x80000000u) ? (o & 0x7fffffffu) : ~o;
    return __builtin_bit_cast(float, u);
}

// MFMA operand vectors.
typedef __attribute__((__vector_size__(8 * sizeof(short)))) short bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float floatx4;

}  // namespace wmi

#define WMI_HIP(call)                                                                  \
    do {                                                                               \
        hipError_t e_ = (call);                                                        \
        if (e_ != hipSuccess)                                                          \
            throw ::wmi::DeviceError(std::string(#call) + ": " + hipGetErrorString(e_)); \
    } while (0)

namespace wmi {
struct DeviceError : std::runtime_error {
    using std::runtime_error::runtime_error;
};
struct ArgError : std::runtime_error {
    int code;
    ArgError(int c, const std::string& m) : std::runtime_error(m), code(c) {}
};
}  // namespace wmi
