// Elementwise parts of a gated (SwiGLU) FFN, whose three projections run
// through the row-typed GEMM: H = silu(Z_g) . Z_u forward, and backward
// dZ_g = dH . Z_u . silu'(Z_g), dZ_u = dH . silu(Z_g); plus the sum of the
// two activation gradients dX = dX_g + dX_u; and the forward from a merged
// gate/up projection's output (gate and up interleaved in 8-feature chunks).  SiLU is z sigma(z) with the
// logistic sigma from the hardware exp2 and reciprocal (about 1 ulp each),
// and sigma'(z) = sigma (1 - sigma).  Every kernel streams 16 bytes per
// thread per operand: HBM-bound, a grid-stride loop over n / 8 (bf16) or
// n / 4 (fp32) vectors.
#include "common.hpp"
#include "kernels.hpp"

namespace starq {

namespace {

template <typename T> struct Vec;
template <> struct Vec<uint16_t> {
  static constexpr int N = 8;
  __device__ static void load(const void* p, int64_t v, float (&f)[8]) {
    const uint4 w = reinterpret_cast<const uint4*>(p)[v];
    const uint32_t u[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f[2 * i] = bf16_to_f32(static_cast<uint16_t>(u[i] & 0xffffu));
      f[2 * i + 1] = bf16_to_f32(static_cast<uint16_t>(u[i] >> 16));
    }
  }
  __device__ static void store(void* p, int64_t v, const float (&f)[8]) {
    uint32_t u[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      u[i] = static_cast<uint32_t>(f32_to_bf16(f[2 * i])) | (static_cast<uint32_t>(f32_to_bf16(f[2 * i + 1])) << 16);
    reinterpret_cast<uint4*>(p)[v] = make_uint4(u[0], u[1], u[2], u[3]);
  }
};
template <> struct Vec<float> {
  static constexpr int N = 4;
  __device__ static void load(const void* p, int64_t v, float (&f)[4]) {
    const float4 w = reinterpret_cast<const float4*>(p)[v];
    f[0] = w.x; f[1] = w.y; f[2] = w.z; f[3] = w.w;
  }
  __device__ static void store(void* p, int64_t v, const float (&f)[4]) {
    reinterpret_cast<float4*>(p)[v] = make_float4(f[0], f[1], f[2], f[3]);
  }
};

template <typename T>
__global__ __launch_bounds__(256) void swiglu_fwd_kernel(int64_t nv, const void* __restrict__ zg,
                                                         const void* __restrict__ zu, void* __restrict__ h) {
  constexpr int N = Vec<T>::N;
  for (int64_t v = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; v < nv;
       v += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    float g[N], u[N], o[N];
    Vec<T>::load(zg, v, g);
    Vec<T>::load(zu, v, u);
#pragma unroll
    for (int i = 0; i < N; ++i) o[i] = g[i] * sigmoid_fast(g[i]) * u[i];
    Vec<T>::store(h, v, o);
  }
}

// Gate and up interleaved in 8-feature chunks (the merged projection's
// layout): feature f's gate at column 16 (f / 8) + f % 8 of a 2F-wide row,
// its up value 8 columns on.  Vector v covers features N v .. N v + N - 1 of
// the flattened [M, F] output (N = 8 bf16 or 4 fp32; F a multiple of 8, so a
// vector never leaves its chunk).
template <typename T>
__global__ __launch_bounds__(256) void swiglu_merged_kernel(int64_t nv, int64_t F, const void* __restrict__ zgu,
                                                            void* __restrict__ h) {
  constexpr int N = Vec<T>::N;
  for (int64_t v = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; v < nv;
       v += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const int64_t e = v * N, row = e / F, f = e - row * F;
    const int64_t g_el = row * 2 * F + 16 * (f / 8) + f % 8;  // element index of the gate values
    float g[N], u[N], o[N];
    Vec<T>::load(zgu, g_el / N, g);
    Vec<T>::load(zgu, (g_el + 8) / N, u);
#pragma unroll
    for (int i = 0; i < N; ++i) o[i] = g[i] * sigmoid_fast(g[i]) * u[i];
    Vec<T>::store(h, v, o);
  }
}

template <typename T>
__global__ __launch_bounds__(256) void swiglu_bwd_kernel(int64_t nv, const void* __restrict__ dh,
                                                         const void* __restrict__ zg, const void* __restrict__ zu,
                                                         void* __restrict__ dzg, void* __restrict__ dzu) {
  constexpr int N = Vec<T>::N;
  for (int64_t v = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; v < nv;
       v += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    float d[N], g[N], u[N], og[N], ou[N];
    Vec<T>::load(dh, v, d);
    Vec<T>::load(zg, v, g);
    Vec<T>::load(zu, v, u);
#pragma unroll
    for (int i = 0; i < N; ++i) {
      const float s = sigmoid_fast(g[i]);
      const float silu = g[i] * s;
      og[i] = d[i] * u[i] * (s + silu * (1.0f - s));
      ou[i] = d[i] * silu;
    }
    Vec<T>::store(dzg, v, og);
    Vec<T>::store(dzu, v, ou);
  }
}

template <typename T>
__global__ __launch_bounds__(256) void add_kernel(int64_t nv, const void* a, const void* b, void* out) {
  constexpr int N = Vec<T>::N;
  for (int64_t v = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; v < nv;
       v += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    float x[N], y[N];
    Vec<T>::load(a, v, x);
    Vec<T>::load(b, v, y);
#pragma unroll
    for (int i = 0; i < N; ++i) x[i] += y[i];
    Vec<T>::store(out, v, x);
  }
}

int blocks_for(int64_t nv) {
  const int64_t b = (nv + 255) / 256;
  return static_cast<int>(b < 1 ? 1 : (b > 8192 ? 8192 : b));
}

}  // namespace

hipError_t launch_swiglu_fwd(int64_t n, int elem, const void* zg, const void* zu, void* h,
                             hipStream_t stream) {
  if (elem == 1) {
    const int64_t nv = n / 8;
    hipLaunchKernelGGL(swiglu_fwd_kernel<uint16_t>, dim3(blocks_for(nv)), dim3(256), 0, stream, nv, zg, zu, h);
  } else {
    const int64_t nv = n / 4;
    hipLaunchKernelGGL(swiglu_fwd_kernel<float>, dim3(blocks_for(nv)), dim3(256), 0, stream, nv, zg, zu, h);
  }
  return hipGetLastError();
}

hipError_t launch_swiglu_merged(int64_t M, int64_t F, int elem, const void* zgu, void* h, hipStream_t stream) {
  const int64_t n = M * F;
  if (elem == 1) {
    const int64_t nv = n / 8;
    hipLaunchKernelGGL(swiglu_merged_kernel<uint16_t>, dim3(blocks_for(nv)), dim3(256), 0, stream, nv, F, zgu, h);
  } else {
    const int64_t nv = n / 4;
    hipLaunchKernelGGL(swiglu_merged_kernel<float>, dim3(blocks_for(nv)), dim3(256), 0, stream, nv, F, zgu, h);
  }
  return hipGetLastError();
}

hipError_t launch_swiglu_bwd(int64_t n, int elem, const void* dh, const void* zg, const void* zu, void* dzg,
                             void* dzu, hipStream_t stream) {
  if (elem == 1) {
    const int64_t nv = n / 8;
    hipLaunchKernelGGL(swiglu_bwd_kernel<uint16_t>, dim3(blocks_for(nv)), dim3(256), 0, stream, nv, dh, zg, zu,
                       dzg, dzu);
  } else {
    const int64_t nv = n / 4;
    hipLaunchKernelGGL(swiglu_bwd_kernel<float>, dim3(blocks_for(nv)), dim3(256), 0, stream, nv, dh, zg, zu, dzg,
                       dzu);
  }
  return hipGetLastError();
}

hipError_t launch_add(int64_t n, int elem, const void* a, const void* b, void* out, hipStream_t stream) {
  if (elem == 1) {
    const int64_t nv = n / 8;
    hipLaunchKernelGGL(add_kernel<uint16_t>, dim3(blocks_for(nv)), dim3(256), 0, stream, nv, a, b, out);
  } else {
    const int64_t nv = n / 4;
    hipLaunchKernelGGL(add_kernel<float>, dim3(blocks_for(nv)), dim3(256), 0, stream, nv, a, b, out);
  }
  return hipGetLastError();
}

}  // namespace starq
