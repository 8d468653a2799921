// Decode-step projection for few rows (one new token per sequence, M <= 64).
//
// Single-token FFN decode is a matrix-vector problem bound by weight
// bandwidth (Sec. 4.2 notes decode needs its own implementation; Sec. 5.3).
// The batched kernel's per-type gathering would read a shared diagonal block
// once per row type present; here every weight block that some row's
// support reaches is streamed exactly once per step instead, and rows whose
// support skips the block multiply zeros.
//
// Grid: (column tiles of 64 outputs within an output group j) x (K chunks of
// 128 inputs within an input group g).  A workgroup
//  1. decides which of the M rows need block (g, j): k = g in B(t_b, j);
//     if none does, the chunk is skipped and its weights are never read;
//  2. stages its rows' inputs (masked per row) and the 128 x 64 weight tile
//     (transposed in registers) in LDS;
//  3. multiplies with v_mfma_f32_32x32x16_bf16 (64 x 64 x 128 per tile);
//  4. writes an fp32 partial, then counts itself done on the column tile's
//     counter.  The last workgroup to finish a column tile sums the partials
//     of its non-skipped chunks in chunk order (deterministic), adds the
//     bias, and applies the phase's epilogue: H = bf16(act(z)) for the up
//     projection; h += z (or h = z), a = bf16(h) for the down projection.
// There is no waiting on other workgroups, so no workgroup can stall.
#include "common.hpp"
#include "kernels.hpp"

namespace starq {

namespace {

constexpr int kThreads = 256;
constexpr int TN = kDecodeTileN;    // 64 output columns
constexpr int TKc = kDecodeChunkK;  // 128 inputs
constexpr int MR = kDecodeMaxRows;  // 64 rows
constexpr int kRowBytes = TKc * 2 + 16;  // 272

__device__ __forceinline__ bool in_support(int law, int i, int j, int k) {
  return law == 1 || k == i || k == j;
}

__device__ __forceinline__ uint32_t word_of(const uint4& r, int w) {
  return w == 0 ? r.x : (w == 1 ? r.y : (w == 2 ? r.z : r.w));
}

__global__ __launch_bounds__(kThreads) void decode_phase_kernel(const DecodePhase p) {
  __shared__ __attribute__((aligned(16))) char As[MR * kRowBytes];
  __shared__ __attribute__((aligned(16))) char Bs[TN * kRowBytes];
  __shared__ int32_t need_s[MR];
  __shared__ int32_t any_g[kMaxQGroups];
  __shared__ int32_t last_s;

  const int tid = threadIdx.x;
  const int ct = blockIdx.x;
  const int kc = blockIdx.y;
  int j = 0;
  while (ct >= p.NTp[j + 1]) ++j;
  int g = 0;
  while (kc >= p.KCp[g + 1]) ++g;
  const int32_t n0 = p.R[j] + (ct - p.NTp[j]) * TN;
  const int32_t nend = p.R[j + 1];
  const int32_t k0 = p.S[g] + (kc - p.KCp[g]) * TKc;
  const int32_t kend = p.S[g + 1];

  if (tid < MR) need_s[tid] = (tid < p.M) && in_support(p.law, p.types[tid], j, g);
  const int any = __syncthreads_or(tid < MR ? need_s[tid] : 0);

  if (any) {
    // stage the rows' inputs: row r = tid/16 + 16u, 16-byte chunk tid%16
    uint4 ra[4];
    const int kq = (tid & 15) * 8;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int r = (tid >> 4) + 16 * u;
      if (need_s[r] && k0 + kq < kend)
        ra[u] = *reinterpret_cast<const uint4*>(p.A + static_cast<int64_t>(r) * p.K + k0 + kq);
      else
        ra[u] = make_uint4(0, 0, 0, 0);
    }
    // stage the weight tile: rows k0 + 4 kb + e, columns n0 + 8 cb .. +8
    uint4 rw[4];
    const int cb = tid & 7;
    const int kb = tid >> 3;
    const int32_t col = n0 + cb * 8;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int32_t k = k0 + kb * 4 + e;
      if (k < kend && col < nend)
        rw[e] = *reinterpret_cast<const uint4*>(p.W + static_cast<int64_t>(k) * p.N + col);
      else
        rw[e] = make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
      *reinterpret_cast<uint4*>(As + ((tid >> 4) + 16 * u) * kRowBytes + (tid & 15) * 16) = ra[u];
#pragma unroll
    for (int v = 0; v < 8; ++v) {
      const int w = v >> 1, sh = (v & 1) * 16;
      uint2 piece;
      piece.x = ((word_of(rw[0], w) >> sh) & 0xffffu) | (((word_of(rw[1], w) >> sh) & 0xffffu) << 16);
      piece.y = ((word_of(rw[2], w) >> sh) & 0xffffu) | (((word_of(rw[3], w) >> sh) & 0xffffu) << 16);
      *reinterpret_cast<uint2*>(Bs + (cb * 8 + v) * kRowBytes + kb * 8) = piece;
    }
    __syncthreads();

    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int lr = lane & 31, lh = lane >> 5;
    f32x16_t acc;
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[e] = 0.f;
    if (wm * 32 < p.M) {
      const char* a_base = As + (wm * 32 + lr) * kRowBytes + lh * 16;
      const char* b_base = Bs + (wn * 32 + lr) * kRowBytes + lh * 16;
#pragma unroll
      for (int s = 0; s < TKc / 16; ++s) {
        const uint4 a = *reinterpret_cast<const uint4*>(a_base + s * 32);
        const uint4 b = *reinterpret_cast<const uint4*>(b_base + s * 32);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                      __builtin_bit_cast(bf16x8_t, b), acc, 0, 0, 0);
      }
      const int32_t n = n0 + wn * 32 + lr;
      if (n < nend) {
        float* part = p.partial + static_cast<int64_t>(kc) * MR * p.N;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int r = wm * 32 + 8 * (e >> 2) + 4 * lh + (e & 3);
          if (r < p.M) part[static_cast<int64_t>(r) * p.N + n] = acc[e];
        }
      }
    }
  }

  // publish this chunk, then let the last workgroup of the column tile reduce
  __threadfence();
  __syncthreads();
  if (tid == 0) {
    const int nk = gridDim.y;
    const int old = atomicAdd(&p.counters[ct], 1);
    last_s = (old == nk - 1);
  }
  __syncthreads();
  if (!last_s) return;
  __threadfence();
  if (tid == 0) p.counters[ct] = 0;  // ready for the next launch
  if (tid < p.q) {
    int a = 0;
    for (int b = 0; b < p.M; ++b) a |= in_support(p.law, p.types[b], j, tid);
    any_g[tid] = a;
  }
  __syncthreads();

  const int nk = gridDim.y;
  for (int idx = tid; idx < p.M * TN; idx += kThreads) {
    const int r = idx / TN;
    const int32_t n = n0 + idx % TN;
    if (n >= nend) continue;
    float z = 0.f;
    int gg = 0;
    for (int c = 0; c < nk; ++c) {
      while (c >= p.KCp[gg + 1]) ++gg;
      if (!any_g[gg]) continue;
      // a chunk that ran but had no row needing it for this row still wrote
      // zeros for that row
      z += __builtin_nontemporal_load(p.partial + (static_cast<int64_t>(c) * MR + r) * p.N + n);
    }
    if (p.bias) z += p.bias[n];
    const int64_t o = static_cast<int64_t>(r) * p.N + n;
    if (p.mode == 0) {
      p.out_bf16[o] = f32_to_bf16(act_fwd(p.act, z));
    } else {
      const float hv = p.residual ? p.h[o] + z : z;
      p.h[o] = hv;
      if (p.out_bf16) p.out_bf16[o] = f32_to_bf16(hv);
      if (p.Y) store_out(p.Y, p.ydtype, o, hv);
    }
  }
}

__global__ void decode_init_kernel(const uint16_t* __restrict__ X, int64_t n, float* __restrict__ h,
                                   uint16_t* __restrict__ xb, int32_t* __restrict__ counters,
                                   int n_counters) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const uint16_t v = X[i];
    h[i] = bf16_to_f32(v);
    xb[i] = v;
  }
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n_counters; i += gridDim.x * blockDim.x)
    counters[i] = 0;
}

}  // namespace

hipError_t launch_decode_init(const uint16_t* X, int64_t n, float* h, uint16_t* xb,
                              int32_t* counters, int n_counters, hipStream_t stream) {
  hipLaunchKernelGGL(decode_init_kernel, dim3(64), dim3(256), 0, stream, X, n, h, xb, counters,
                     n_counters);
  return hipGetLastError();
}

hipError_t launch_decode_phase(const DecodePhase& p, hipStream_t stream) {
  dim3 grid(p.NTp[p.q], p.KCp[p.q]);
  hipLaunchKernelGGL(decode_phase_kernel, grid, dim3(kThreads), 0, stream, p);
  return hipGetLastError();
}

}  // namespace starq
