// Bias gradient of the weight-gradient path: column sums of dY over the
// rows of valid type, in fixed row chunks (the chunks are then summed in
// order), so dbias does not depend on timing.
#include "common.hpp"
#include "kernels.hpp"

namespace starq {

namespace {

// part[c][n] = sum over rows [c * chunk, (c + 1) * chunk) of the rows of
// valid type of the bf16 (or fp32) matrix src [M][N].  When every row has a valid type
// (offsets[q] == M) the rows are taken in their own order (contiguous
// reads); otherwise in type-sorted order, row perm[position] for positions
// below offsets[q].  A block covers 8 * (256 / RL) columns: thread (g, r)
// adds 8 columns (one 16-byte load per row) over rows r, r + RL, ... of the
// chunk in order, then the RL row lanes are added in order through LDS, so
// the result does not depend on scheduling.  The rows are loaded 8 at a time
// before they are added (one load in flight per thread left the kernel
// waiting on memory latency).  RL = 16 for narrow matrices: twice the
// blocks, half the rows per thread.
template <typename T, int RL>
__global__ __launch_bounds__(256) void column_sum_kernel(const T* __restrict__ src, int32_t N,
                                                         const int32_t* __restrict__ perm,
                                                         const int32_t* __restrict__ offsets, int q,
                                                         int32_t M, int32_t chunk, float* __restrict__ part) {
  constexpr int CG = 256 / RL, BC = 8 * CG;  // column groups and columns per block
  __shared__ float red[RL][BC + 4];
  const int32_t rows = offsets[q];
  const bool natural = rows == M;
  const int32_t c = blockIdx.y;
  const int g = threadIdx.x % CG, rl = threadIdx.x / CG;
  const int32_t n0 = blockIdx.x * BC + 8 * g;
  const int32_t r0 = c * chunk, r1 = min(rows, r0 + chunk);
  float sum[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (n0 < N) {
    constexpr int U = 8;  // rows in flight per thread
    for (int32_t rb = r0 + rl; rb < r1; rb += RL * U) {
      int32_t row[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int32_t r = rb + RL * u;
        row[u] = r < r1 ? (natural ? r : perm[r]) : -1;
      }
      if constexpr (sizeof(T) == 2) {
        uint4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u)
          v[u] = row[u] >= 0 ? *reinterpret_cast<const uint4*>(src + static_cast<int64_t>(row[u]) * N + n0)
                             : make_uint4(0, 0, 0, 0);
#pragma unroll
        for (int u = 0; u < U; ++u) {
          if (row[u] < 0) continue;
          sum[0] += bf16_to_f32(v[u].x & 0xffffu); sum[1] += bf16_to_f32(v[u].x >> 16);
          sum[2] += bf16_to_f32(v[u].y & 0xffffu); sum[3] += bf16_to_f32(v[u].y >> 16);
          sum[4] += bf16_to_f32(v[u].z & 0xffffu); sum[5] += bf16_to_f32(v[u].z >> 16);
          sum[6] += bf16_to_f32(v[u].w & 0xffffu); sum[7] += bf16_to_f32(v[u].w >> 16);
        }
      } else {
        float4 a[U], b[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const bool ok = row[u] >= 0;
          const float* pr = src + static_cast<int64_t>(ok ? row[u] : 0) * N + n0;
          a[u] = ok ? *reinterpret_cast<const float4*>(pr) : make_float4(0.f, 0.f, 0.f, 0.f);
          b[u] = ok ? *reinterpret_cast<const float4*>(pr + 4) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
          if (row[u] < 0) continue;
          sum[0] += a[u].x; sum[1] += a[u].y; sum[2] += a[u].z; sum[3] += a[u].w;
          sum[4] += b[u].x; sum[5] += b[u].y; sum[6] += b[u].z; sum[7] += b[u].w;
        }
      }
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) red[rl][8 * g + e] = sum[e];
  __syncthreads();
  if (threadIdx.x < BC) {
    const int32_t n = blockIdx.x * BC + threadIdx.x;
    if (n < N) {
      float t = 0.f;
#pragma unroll
      for (int k = 0; k < RL; ++k) t += red[k][threadIdx.x];
      part[static_cast<int64_t>(c) * N + n] = t;
    }
  }
}

// out[n] = the sum of part[c][n] over c < nparts, for few outputs and many
// parts (the chunk sums above): a block takes 32 consecutive outputs; thread
// (g, j) adds parts g, g + 8, g + 16, ... of output j in that order, eight
// loads in flight, and the eight group sums are added in order through LDS.
__global__ __launch_bounds__(256) void sum_chunks_kernel(const float* __restrict__ part, int nparts,
                                                         int32_t n, float* __restrict__ out) {
  __shared__ float red[8][32];
  const int j = threadIdx.x & 31, g = threadIdx.x >> 5;
  const int32_t col = blockIdx.x * 32 + j;
  float acc = 0.f;
  if (col < n) {
    for (int c0 = g; c0 < nparts; c0 += 64) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int c = c0 + 8 * u;
        v[u] = c < nparts ? part[static_cast<int64_t>(c) * n + col] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (c0 + 8 * u < nparts) acc += v[u];
    }
  }
  red[g][j] = acc;
  __syncthreads();
  if (g == 0 && col < n) {
    float t = 0.f;
#pragma unroll
    for (int k = 0; k < 8; ++k) t += red[k][j];
    out[col] = t;
  }
}

template <typename T>
hipError_t launch_colsum(const T* src, int32_t N, const int32_t* perm, const int32_t* offsets, int q,
                         int32_t M, int32_t chunk, int nchunks, float* part, hipStream_t stream) {
  if (N <= 1536) {
    hipLaunchKernelGGL((column_sum_kernel<T, 16>), dim3((N + 127) / 128, nchunks), dim3(256), 0, stream, src,
                       N, perm, offsets, q, M, chunk, part);
  } else {
    hipLaunchKernelGGL((column_sum_kernel<T, 8>), dim3((N + 255) / 256, nchunks), dim3(256), 0, stream, src,
                       N, perm, offsets, q, M, chunk, part);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_column_sum(const uint16_t* src, int32_t N, const int32_t* perm, const int32_t* offsets,
                             int q, int32_t M, int32_t chunk, int nchunks, float* part, hipStream_t stream) {
  return launch_colsum(src, N, perm, offsets, q, M, chunk, nchunks, part, stream);
}

hipError_t launch_column_sum_f32(const float* src, int32_t N, const int32_t* perm, const int32_t* offsets,
                                 int q, int32_t M, int32_t chunk, int nchunks, float* part, hipStream_t stream) {
  return launch_colsum(src, N, perm, offsets, q, M, chunk, nchunks, part, stream);
}

hipError_t launch_sum_chunks(const float* part, int nparts, int32_t n, float* out, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(sum_chunks_kernel, dim3((n + 31) / 32), dim3(256), 0, stream, part, nparts, n, out);
  return hipGetLastError();
}

}  // namespace starq
