// Device-side helpers shared by the gfx950 kernels of libstarq.
#pragma once

#include <atomic>

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace starq {

constexpr int kMaxQ = 64;

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// bfloat16 storage type: raw bits.
struct bf16 {
  uint16_t bits;
};

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// Round-to-nearest-even from binary32 (NaN kept quiet).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((u >> 16) | 0x40);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

// ---- activations -----------------------------------------------------------
// One GELU for every kernel (GEMM epilogues and the decode kernels), with
// explicit approximations whose error bounds are stated and tested.

enum Act : int { kActNone = 0, kActGelu = 1, kActGeluTanh = 2 };

constexpr float kLog2e = 1.4426950408889634f;

// tanh(u) = 1 - 2 / (1 + exp(2u)); the absolute error stays near 1e-7 over
// the whole range (saturating to +-1), which is what the tanh-form GELU needs.
__device__ __forceinline__ float tanh_fast(float u) {
  return 1.0f - 2.0f * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(2.0f * kLog2e * u));
}

// Exact-form GELU, z Phi(z) = z (1 + erf(z / sqrt 2)) / 2, with erf from
// Abramowitz & Stegun 7.1.28: erf(x) = 1 - (1 + a1 x + ... + a6 x^6)^-16 for
// x >= 0, |error| <= 3e-7.  With r = p(|z| / sqrt 2)^-16 the identity
// z Phi(z) = max(z, 0) - |z| r / 2 holds for either sign of z; the 1 / sqrt 2
// goes into the coefficients (a_k 2^(-k/2)) and the 1 / 2 too, by scaling
// the whole polynomial by 2^(1/16).  So: six FMAs, four squarings, one
// reciprocal, a max and an FMA, and no exponential.  Error in fp32 at most
// 1e-6 + 2^-22 |GELU(z)| for every z (the test of the device activations
// checks this element by element over [-12, 12] and the tails); p^16
// overflows to infinity for large |z|, where r = 0 is the right limit.
__device__ __forceinline__ float gelu_erf(float z) {
  const float az = fabsf(z);
  float p = 5.6212996640e-06f;
  p = p * az + 5.1055209008e-05f;
  p = p * az + 3.9686137011e-05f;
  p = p * az + 3.4227392389e-03f;
  p = p * az + 2.2076998457e-02f;
  p = p * az + 5.2075163037e-02f;
  p = p * az + 1.0442737824e+00f;
  p *= p;
  p *= p;
  p *= p;
  p *= p;
  return fmaf(-az, __builtin_amdgcn_rcpf(p), fmaxf(z, 0.0f));
}

// Tanh form 0.5 z (1 + tanh(sqrt(2/pi) (z + 0.044715 z^3))): error at most
// 1e-6 + 2^-22 |value|.
// The logistic function for SiLU (z sigma(z)): the hardware exp2 and
// reciprocal, about 1 ulp each.  Every SwiGLU kernel uses this one.
__device__ __forceinline__ float sigmoid_fast(float z) {
  return __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-z * 1.4426950408889634f));
}

__device__ __forceinline__ float act_apply(int act, float z) {
  if (act == kActGelu) return gelu_erf(z);
  if (act == kActGeluTanh) {
    const float u = 0.79788456080286536f * (z + 0.044715f * z * z * z);
    return 0.5f * z * (1.0f + tanh_fast(u));
  }
  return z;
}

// d act / dz.  Erf form Phi(z) + z phi(z), Phi through A&S 7.1.26 at
// x = |z| / sqrt 2; its factor exp(-x^2) = exp(-z^2 / 2) is also
// sqrt(2 pi) phi(z), so one exponential serves both terms.  Error at most
// 1e-6.  Tanh form: error at most 5e-6 (the 1 - t^2 factor loses digits
// where tanh saturates).
__device__ __forceinline__ float act_deriv(int act, float z) {
  if (act == kActGelu) {
    const float x = fabsf(z) * 0.70710678118654752f;
    const float t = __builtin_amdgcn_rcpf(1.0f + 0.3275911f * x);
    float poly = 1.061405429f;
    poly = poly * t - 1.453152027f;
    poly = poly * t + 1.421413741f;
    poly = poly * t - 0.284496736f;
    poly = poly * t + 0.254829592f;
    poly *= t;
    const float e = __builtin_amdgcn_exp2f(-(x * x) * kLog2e);
    const float tail = 0.5f * poly * e;  // 1 - Phi(|z|)
    return fmaf(z * 0.39894228040143268f, e, z >= 0.0f ? 1.0f - tail : tail);
  }
  if (act == kActGeluTanh) {
    const float u = 0.79788456080286536f * (z + 0.044715f * z * z * z);
    const float t = tanh_fast(u);
    const float du = 0.79788456080286536f * (1.0f + 0.134145f * z * z);
    return 0.5f * (1.0f + t) + 0.5f * z * (1.0f - t * t) * du;
  }
  return 1.0f;
}

// ---- element access ------------------------------------------------------

template <typename T> struct Elem;
template <> struct Elem<float> {
  static constexpr int kVec = 4;  // elements per 16 bytes
  __device__ static float load(const float* p, int64_t i) { return p[i]; }
};
template <> struct Elem<bf16> {
  static constexpr int kVec = 8;
  __device__ static float load(const bf16* p, int64_t i) { return bf16_to_f32(p[i].bits); }
};

// Store one value into an output of runtime dtype (0 = f32, 1 = bf16).
__device__ __forceinline__ void store_out(void* base, int dtype, int64_t idx, float v) {
  if (dtype == 0)
    static_cast<float*>(base)[idx] = v;
  else
    static_cast<uint16_t*>(base)[idx] = f32_to_bf16(v);
}

__device__ __forceinline__ float load_in(const void* base, int dtype, int64_t idx) {
  if (dtype == 0) return static_cast<const float*>(base)[idx];
  return bf16_to_f32(static_cast<const uint16_t*>(base)[idx]);
}


// Raises a kernel's dynamic-LDS limit to `bytes` once per device: the
// attribute belongs to the function on the current device, so `done`
// (one per kernel) records the devices already set.
inline hipError_t ensure_lds_limit(const void* fn, std::atomic<unsigned long long>& done, int bytes) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return hipErrorInvalidDevice;
  const unsigned long long bit = dev < 64 ? (1ull << dev) : 0ull;
  if (bit && (done.load(std::memory_order_relaxed) & bit)) return hipSuccess;
  const hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (e == hipSuccess && bit) done.fetch_or(bit, std::memory_order_relaxed);
  return e;
}

}  // namespace starq
