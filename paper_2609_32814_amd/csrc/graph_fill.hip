// The output blocks of the graph law (Sec. "Graph Products with Exact Cost")
// that no row's support reaches.  Under Q_G a type-i row's slots are its
// vertex slot i and the edge slots (i, j) of its out-edges; an output group
// j != i without the edge i -> j is not a slot of the row, so its product is
// zero: the forward writes act(bias) there (and the bias into Z), the
// activation gradient writes zeros into such input groups.  The GEMM never
// visits these blocks (its tile passes leave them out), so this kernel and
// the GEMM write disjoint parts of the output.  A plain stream over the
// plan's positions: one thread per 8 consecutive outputs of one row (group
// widths are multiples of 8); rows of out-of-range type are not written.
#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"

namespace starq {

namespace {

__global__ __launch_bounds__(256) void graph_fill_kernel(const GemmParams p, int mode) {
  const int32_t W = mode == kModeFwd ? p.N : p.K;  // output row width
  const int32_t* G = mode == kModeFwd ? p.R : p.S;  // output group starts
  const int32_t per_row = W / 8;
  // the rows of valid type, in the plan's type-sorted order: position pos
  // holds row perm[pos] of the class whose offsets bracket pos
  const int32_t rows = p.offsets[p.q];
  const int64_t total = static_cast<int64_t>(rows) * per_row;
  for (int64_t u = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; u < total;
       u += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const int32_t pos = static_cast<int32_t>(u / per_row);
    const int32_t c0 = static_cast<int32_t>(u % per_row) * 8;
    int ti = 0;
    while (ti + 1 < p.q && pos >= p.offsets[ti + 1]) ++ti;
    int j = 0;
    while (j + 1 < p.q && c0 >= G[j + 1]) ++j;
    if (j == ti || ((p.adj[ti] >> j) & 1ull)) continue;  // a slot: the GEMM writes it
    const int32_t row = p.perm[pos];
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = (mode == kModeFwd && p.bias) ? p.bias[c0 + e] : 0.f;
    const int64_t o = static_cast<int64_t>(row) * W + c0;
    if (mode == kModeFwd && p.Z) {
#pragma unroll
      for (int e = 0; e < 8; ++e) store_out(p.Z, p.ydtype, o + e, v[e]);
    }
    if (mode == kModeFwd) {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = act_apply(p.act, v[e]);
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) store_out(p.Y, p.ydtype, o + e, v[e]);
  }
}

}  // namespace

hipError_t launch_graph_fill(int mode, const GemmParams& p, hipStream_t stream) {
  const int32_t W = mode == kModeFwd ? p.N : p.K;
  const int64_t total = static_cast<int64_t>(p.M) * (W / 8);
  const int blocks = static_cast<int>(std::min<int64_t>(4096, (total + 255) / 256 + 1));
  hipLaunchKernelGGL(graph_fill_kernel, dim3(blocks), dim3(256), 0, stream, p, mode);
  return hipGetLastError();
}

}  // namespace starq
