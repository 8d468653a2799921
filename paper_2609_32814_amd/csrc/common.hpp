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
// Exact GELU uses the ROCm device library's erff; the tanh form its tanhf.

enum Act : int { kActNone = 0, kActGelu = 1, kActGeluTanh = 2 };

__device__ __forceinline__ float act_fwd(int act, float z) {
  if (act == kActGelu) return 0.5f * z * (1.0f + erff(z * 0.70710678118654752f));
  if (act == kActGeluTanh) {
    float u = 0.79788456080286536f * (z + 0.044715f * z * z * z);
    return 0.5f * z * (1.0f + tanhf(u));
  }
  return z;
}

__device__ __forceinline__ float act_grad(int act, float z) {
  if (act == kActGelu)
    return 0.5f * (1.0f + erff(z * 0.70710678118654752f)) +
           z * 0.39894228040143268f * __expf(-0.5f * z * z);
  if (act == kActGeluTanh) {
    float u = 0.79788456080286536f * (z + 0.044715f * z * z * z);
    float t = tanhf(u);
    float du = 0.79788456080286536f * (1.0f + 0.134145f * z * z);
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
