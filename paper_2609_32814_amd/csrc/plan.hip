// Type plan: the per-type row index sets I_i of Alg. 1 as one stable
// permutation of the rows grouped by type, plus per-type offsets.
//
// Up to 64 Ki rows: many workgroups (type_plan_wide_kernel below).  Longer
// type vectors: one workgroup of 1024 threads (16 wavefronts).  All threads first copy the
// type vector into LDS as 16-bit values with independent coalesced loads (one round
// trip to memory instead of one per window), for up to 64 Ki rows; longer
// vectors are read from memory in the passes below.  The rows are cut into
// 16 contiguous chunks, one per wavefront; a wavefront walks its chunk in
// windows of 64 rows.  Lanes holding the same type find each other with
// ballots over the type bits (a match-any), so each window costs O(log q)
// ballots and no atomics.  Pass 1 counts rows per (wavefront, type); one
// wavefront scans the counts into exclusive bases with lane shuffles; pass 2
// re-walks the chunks and writes each row at base + rank-within-window,
// which keeps the order of rows of one type (stable).  Rows with a type outside [0, q) go to a
// trailing bucket after all valid rows, so perm stays a permutation and no
// tile ever reads them.
#include "common.hpp"
#include "kernels.hpp"

namespace starq {

namespace {

constexpr int kPlanThreads = 1024;
constexpr int kPlanMaxQ = kMaxQFwd;  // types the plan takes (the forward product's limit)
constexpr int kPlanWaves = kPlanThreads / 64;
constexpr int kPlanLdsRows = 65536;

__device__ __forceinline__ uint64_t match_type(int t, bool valid, int nbits) {
  uint64_t m = __ballot(valid);
  if (!valid) m = ~m;
  for (int bit = 0; bit < nbits; ++bit) {
    const bool set = (t >> bit) & 1;
    const uint64_t b = __ballot(set);
    m &= set ? b : ~b;
  }
  return m;
}

__global__ __launch_bounds__(kPlanThreads) void type_plan_kernel(const int32_t* __restrict__ types,
                                                                 int32_t M, int q, int nbits,
                                                                 int32_t* __restrict__ perm,
                                                                 int32_t* __restrict__ offsets) {
  // counts[w][t], t = q is the out-of-range bucket
  __shared__ int32_t counts[kPlanWaves][kPlanMaxQ + 1];
  __shared__ uint16_t tl[kPlanLdsRows];  // type (or q if out of range) per row
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  for (int i = threadIdx.x; i < kPlanWaves * (kPlanMaxQ + 1); i += kPlanThreads)
    (&counts[0][0])[i] = 0;
  const bool in_lds = M <= kPlanLdsRows;
  if (in_lds) {
    constexpr int kBatch = 8;
    for (int32_t base = 0; base < M; base += kPlanThreads * kBatch) {
      int v[kBatch];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int32_t row = base + u * kPlanThreads + threadIdx.x;
        v[u] = row < M ? types[row] : 0;
      }
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int32_t row = base + u * kPlanThreads + threadIdx.x;
        if (row < M) tl[row] = static_cast<uint16_t>((v[u] >= 0 && v[u] < q) ? v[u] : q);
      }
    }
  }
  __syncthreads();
  auto type_of = [&](int32_t row) -> int {
    if (in_lds) return tl[row];
    const int t = types[row];
    return (t >= 0 && t < q) ? t : q;
  };

  const int32_t chunk = ((M + kPlanWaves - 1) / kPlanWaves + 63) & ~63;
  const int32_t lo = wave * chunk;
  const int32_t hi = min(M, lo + chunk);
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));

  // pass 1: counts
  for (int32_t base = lo; base < hi; base += 64) {
    const int32_t row = base + lane;
    const bool in = row < hi;
    const int t = in ? type_of(row) : 0;
    const uint64_t active = __ballot(in);
    const uint64_t m = match_type(t, t < q, nbits) & active;
    if (in && (m & lt_mask) == 0) counts[wave][t] += __popcll(m);
  }
  __syncthreads();

  // exclusive scan of the counts in (type, wavefront) order, by wavefront 0
  // with lane shuffles, 64 entries a round: the bases per (wavefront, type),
  // and per type the offset (offsets[q]: end of the valid rows)
  if (wave == 0) {
    const int n = (q + 1) * kPlanWaves;
    int32_t carry = 0;
    for (int base = 0; base < n; base += 64) {
      const int e = base + lane;
      const int t = e / kPlanWaves, w = e % kPlanWaves;
      const int32_t c = e < n ? counts[w][t] : 0;
      int32_t incl = c;
#pragma unroll
      for (int d = 1; d < 64; d <<= 1) {
        const int32_t u = __shfl_up(incl, d);
        if (lane >= d) incl += u;
      }
      if (e < n) {
        const int32_t excl = carry + incl - c;
        counts[w][t] = excl;
        if (w == 0) offsets[t] = excl;
      }
      carry += __shfl(incl, 63);
    }
  }
  __syncthreads();

  // pass 2: stable scatter
  for (int32_t base = lo; base < hi; base += 64) {
    const int32_t row = base + lane;
    const bool in = row < hi;
    const int t = in ? type_of(row) : 0;
    const uint64_t active = __ballot(in);
    const uint64_t m = match_type(t, t < q, nbits) & active;
    if (in) {
      const int32_t pos = counts[wave][t] + __popcll(m & lt_mask);
      perm[pos] = row;
    }
    // all lanes have read counts[wave][*] before the leaders advance them
    __builtin_amdgcn_wave_barrier();
    if (in && (m & lt_mask) == 0) counts[wave][t] += __popcll(m);
    __builtin_amdgcn_wave_barrier();
  }
}

// Many-workgroup plan for M <= kPlanLdsRows: workgroup g places rows
// [1024 g, 1024 g + 1024).  Every workgroup reads the whole type vector
// (at most 256 KB, from L2) and counts, per type, all rows and the rows
// before its own range; the type offsets and its own bases follow without
// any cross-workgroup synchronisation.  Its rows then go out in order: the
// rank of a row is the number of rows of its type in earlier wavefronts of
// the workgroup plus those in earlier lanes of its own (ballots), so the
// permutation is stable.  Workgroup 0 writes the offsets.
constexpr int kPlanRowsPerBlock = kPlanThreads;

//
// NT > 0 (q + 1 = NT classes, few types): the counting pass takes one ballot
// per class and window and keeps the counts in wave-uniform registers (no
// LDS atomics); the wavefronts' counts are summed after the pass.  NT = 0:
// any q, a match-any per window and LDS atomics from the leading lanes.
template <int NT>
__global__ __launch_bounds__(kPlanThreads) void type_plan_wide_kernel(const int32_t* __restrict__ types,
                                                                      int32_t M, int q, int nbits,
                                                                      int32_t* __restrict__ perm,
                                                                      int32_t* __restrict__ offsets) {
  __shared__ int32_t total[kPlanMaxQ + 1], before[kPlanMaxQ + 1];
  __shared__ int32_t wcount[kPlanWaves][kPlanMaxQ + 1];
  __shared__ int32_t wtot[kPlanWaves][NT > 0 ? NT : 1], wbef[kPlanWaves][NT > 0 ? NT : 1];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int32_t r0 = blockIdx.x * kPlanRowsPerBlock;
  for (int i = threadIdx.x; i <= q; i += kPlanThreads) total[i] = before[i] = 0;
  for (int i = threadIdx.x; i < kPlanWaves * (kPlanMaxQ + 1); i += kPlanThreads) (&wcount[0][0])[i] = 0;
  __syncthreads();
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  auto cls = [&](int t) { return (t >= 0 && t < q) ? t : q; };
  // per-type counts over all rows and over the rows before r0, a 64-row
  // window per wavefront at a time, 8 windows' loads in flight
  // (NT > 0: the valid classes by ballots on the raw type, the out-of-range
  // class as the rest of the rows counted)
  int32_t cnt[NT > 0 ? NT : 1] = {}, bef[NT > 0 ? NT : 1] = {};
  int32_t all = 0, all_bef = 0;
  constexpr int kBatch = 8;
  for (int32_t base = 0; base < M; base += kPlanThreads * kBatch) {
    int v[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int32_t row = base + u * kPlanThreads + threadIdx.x;
      v[u] = row < M ? types[row] : 0;
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int32_t wbase = base + u * kPlanThreads;  // workgroup-uniform
      if (wbase >= M) break;
      if constexpr (NT > 0) {
        // the windows before r0 are those with wbase < r0 (both multiples of
        // the workgroup's row count): keep the counts reached at r0
        if (wbase == r0) {
#pragma unroll
          for (int k = 0; k < NT - 1; ++k) bef[k] = cnt[k];
          all_bef = all;
        }
      }
      const int32_t wrow = wbase + wave * 64;  // the window's first row (wave-uniform)
      if (wrow >= M) break;
      const int32_t row = wrow + lane;
      const bool in = row < M;
      if constexpr (NT > 0) {
        all += __popcll(__ballot(in));
#pragma unroll
        for (int k = 0; k < NT - 1; ++k) cnt[k] += __popcll(__ballot(in && v[u] == k));
      } else {
        const int t = cls(v[u]);
        const uint64_t active = __ballot(in);
        const uint64_t m = match_type(t, t < q, nbits) & active;
        if (in && (m & lt_mask) == 0) {
          atomicAdd(&total[t], __popcll(m));
          if (wrow < r0) atomicAdd(&before[t], __popcll(m));  // windows never straddle r0
        }
      }
    }
  }
  if constexpr (NT > 0) {
    if (lane == 0) {
      int32_t valid = 0, valid_bef = 0;
#pragma unroll
      for (int k = 0; k < NT - 1; ++k) {
        wtot[wave][k] = cnt[k];
        wbef[wave][k] = bef[k];
        valid += cnt[k];
        valid_bef += bef[k];
      }
      wtot[wave][NT - 1] = all - valid;
      wbef[wave][NT - 1] = all_bef - valid_bef;
    }
  }
  // this workgroup's rows: per-wavefront counts per type
  const int32_t row = r0 + threadIdx.x;
  const bool in = row < M;
  const int t = in ? cls(types[row]) : 0;
  const uint64_t active = __ballot(in);
  const uint64_t m = match_type(t, t < q, nbits) & active;
  if (in && (m & lt_mask) == 0) wcount[wave][t] = __popcll(m);
  __syncthreads();
  if constexpr (NT > 0) {
    if (threadIdx.x < NT) {
      int32_t a = 0, b = 0;
      for (int w = 0; w < kPlanWaves; ++w) {
        a += wtot[w][threadIdx.x];
        b += wbef[w][threadIdx.x];
      }
      total[threadIdx.x] = a;
      before[threadIdx.x] = b;
    }
    __syncthreads();
  }
  if (in) {
    // offset of type t, the rows of type t before this workgroup and before
    // this wavefront in it, and the lanes below this one
    int32_t pos = 0;
    for (int u = 0; u < t; ++u) pos += total[u];
    pos += before[t];
    for (int w = 0; w < wave; ++w) pos += wcount[w][t];
    pos += __popcll(m & lt_mask);
    perm[pos] = row;
  }
  if (blockIdx.x == 0 && threadIdx.x <= q) {
    int32_t o = 0;
    for (int u = 0; u < static_cast<int>(threadIdx.x); ++u) o += total[u];
    offsets[threadIdx.x] = o;
  }
}

__global__ void count_bad_types_kernel(const int32_t* __restrict__ types, int64_t M, int q,
                                       unsigned long long* __restrict__ n_bad) {
  unsigned long long local = 0;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < M;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int t = types[i];
    local += (t < 0 || t >= q) ? 1ull : 0ull;
  }
  for (int off = 32; off > 0; off >>= 1) local += __shfl_down(local, off);
  if ((threadIdx.x & 63) == 0 && local) atomicAdd(n_bad, local);
}

}  // namespace

hipError_t launch_type_plan(const int32_t* types, int64_t M, int q, int32_t* perm,
                            int32_t* offsets, hipStream_t stream) {
  int nbits = 0;
  while ((1 << nbits) < q + 1) ++nbits;
  if (M > 0 && M <= kPlanLdsRows) {
    const unsigned blocks = static_cast<unsigned>((M + kPlanRowsPerBlock - 1) / kPlanRowsPerBlock);
    const int32_t m32 = static_cast<int32_t>(M);
    switch (q + 1) {
#define STARQ_PLAN_NT(nt)                                                                        \
  case nt:                                                                                       \
    hipLaunchKernelGGL(type_plan_wide_kernel<nt>, dim3(blocks), dim3(kPlanThreads), 0, stream, \
                       types, m32, q, nbits, perm, offsets);                                     \
    break;
      STARQ_PLAN_NT(2)
      STARQ_PLAN_NT(3)
      STARQ_PLAN_NT(4)
      STARQ_PLAN_NT(5)
      STARQ_PLAN_NT(9)
#undef STARQ_PLAN_NT
      default:
        hipLaunchKernelGGL(type_plan_wide_kernel<0>, dim3(blocks), dim3(kPlanThreads), 0, stream,
                           types, m32, q, nbits, perm, offsets);
    }
  } else {
    hipLaunchKernelGGL(type_plan_kernel, dim3(1), dim3(kPlanThreads), 0, stream, types,
                       static_cast<int32_t>(M), q, nbits, perm, offsets);
  }
  return hipGetLastError();
}

hipError_t launch_count_bad_types(const int32_t* types, int64_t M, int q,
                                  unsigned long long* n_bad, hipStream_t stream) {
  const int64_t blocks64 = (M + 255) / 256;
  const int blocks = static_cast<int>(blocks64 < 1024 ? (blocks64 > 0 ? blocks64 : 1) : 1024);
  hipLaunchKernelGGL(count_bad_types_kernel, dim3(blocks), dim3(256), 0, stream, types, M, q,
                     n_bad);
  return hipGetLastError();
}

}  // namespace starq
