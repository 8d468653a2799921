// Decode-step projection for few rows (one new token per sequence, M <= 64).
//
// Single-token FFN decode is a matrix-vector problem bound by weight
// bandwidth (Sec. 4.2 notes that decode needs its own implementation;
// Sec. 5.3).  The batched kernel's per-type gathering would read a shared
// diagonal block once per row type present; here every weight block that
// some row's support reaches is streamed exactly once per step, and rows
// whose support skips the block multiply zeros.
//
// A workgroup owns 16 output columns (inside one output group j) over the
// whole K range, so no partial sums cross workgroups and no workgroup ever
// waits on another (a kernel boundary separates dependent phases).  K is cut
// into 32-row slices; a slice is needed when some row's support reaches one
// of its input groups (k in B(t_b, j)).  Each of the 4 wavefronts streams
// every fourth needed slice straight from global memory into LDS with one
// 16-byte-per-lane direct load (32 rows x 32 bytes = 1 KB per slice), all
// issued before any is consumed, so the whole weight tile is in flight at
// once (in passes of up to 128 slices when K is wider than 4096: a wave
// reuses only its own slots, so the passes need no barrier).  The wavefront then reads each slice back with the LDS transpose
// read (two reads give every lane 8 consecutive K values of one column),
// loads the rows' 8-element input pieces (zero where the support skips
// them), and multiplies with v_mfma_f32_16x16x32_bf16.  The four
// wavefronts' partial sums are added in LDS in a fixed order, then the bias,
// activation or residual are applied and the outputs written.
//
// Column tiles are mapped to workgroups so that the four tiles sharing a
// 128-byte line of a weight row run on the same XCD (workgroups are
// dispatched round-robin over the 8 XCDs) and share one L2 fetch.
#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"

namespace starq {

namespace {

constexpr int kThreads = 256;
constexpr int TN = kDecodeTileN;      // 16 output columns
constexpr int SLICE = kDecodeSliceK;  // 32 K rows
constexpr int kRedBytes = 4 * 4 * 64 * 16;  // 4 waves x 4 row blocks x 64 lanes x float4
constexpr int kPassSlices = 128;            // most slices held in LDS at once (128 KB)

typedef short v4i16_t __attribute__((ext_vector_type(4)));
#define STARQ_LDS __attribute__((address_space(3)))

// k in B(i, j): law 0 {i, j}; law 1 every group; law 2 (tensor power of
// the two-group law) every bit of k equal to that bit of i or of j; law 3
// (graph algebra, bit j of adj[i] for the edge i -> j) {i} for j = i, {i, j}
// for an edge, nothing otherwise
__device__ __forceinline__ bool in_support(int law, const uint64_t* adj, int i, int j, int k) {
  if (law == 2) return ((k ^ i) & (k ^ j)) == 0;
  if (law == 3) {
    // graph algebra: B(i,i) = {i}, B(i,j) = {i, j} for an edge i -> j, empty otherwise
    if (j == i) return k == i;
    return ((adj[i] >> j) & 1ull) && (k == i || k == j);
  }
  return law == 1 || k == i || k == j;
}

// the input group of index x: the last g with starts[g] <= x, by binary
// search over the starts (held in LDS: searched from the kernel's argument
// block, every step was a dependent scalar load)
__device__ __forceinline__ int group_of(const int32_t* starts, int q, int32_t x) {
  int lo = 0, hi = q - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (x >= starts[mid]) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

__global__ __launch_bounds__(kThreads) void decode_phase_kernel(const DecodePhase p) {
  extern __shared__ __attribute__((aligned(16))) char lds[];
  __shared__ unsigned long long rowmask_s[kMaxQGroups];
  __shared__ int32_t S_s[kMaxQGroups + 1];
  __shared__ int16_t slices_s[kDecodeMaxK / SLICE];
  __shared__ int32_t wave_cnt_s[4];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;

  // column tile of this workgroup (XCD-aware: 4 consecutive tiles per XCD)
  const int b = blockIdx.x;
  const int xcd = b & 7, s = b >> 3;
  const int ct = 4 * (8 * (s >> 2) + xcd) + (s & 3);
  const int nt_total = p.NTp[p.q];
  if (ct >= nt_total) return;
  int j = 0;
  while (ct >= p.NTp[j + 1]) ++j;
  const int32_t n0 = p.R[j] + (ct - p.NTp[j]) * TN;
  const int32_t nend = p.R[j + 1];

  // the input group starts, searched from LDS below
  for (int i = tid; i <= p.q; i += kThreads) S_s[i] = p.S[i];
  __syncthreads();
  // which rows need block (g, j), per input group g: wave 0 holds one row
  // per lane and takes one ballot per group
  if (wave == 0) {
    // a row whose type lies outside [0, q) has an empty support
    const int t = lane < p.M ? p.types[lane] : -1;
    const bool valid = t >= 0 && t < p.q;
    for (int g = 0; g < p.q; ++g) {
      const unsigned long long m = __ballot(valid && in_support(p.law, p.adj, t, j, g));
      if (lane == 0) rowmask_s[g] = m;
    }
  }
  __syncthreads();
  // needed slices, in K order: one slice per thread a round (256 slices a
  // round), compacted with ballots
  const int nsl = (p.K + SLICE - 1) / SLICE;  // <= kDecodeMaxK / SLICE
  int32_t found = 0;                          // needed slices before this round
  for (int base = 0; base < nsl; base += kThreads) {
    const int sl = base + tid;
    bool need = false;
    if (sl < nsl) {
      for (int piece = 0; piece < SLICE / 8; ++piece) {
        const int32_t k = sl * SLICE + piece * 8;
        if (k < p.K && rowmask_s[group_of(S_s, p.q, k)]) need = true;
      }
    }
    const unsigned long long bal = __ballot(need);
    if (lane == 0) wave_cnt_s[wave] = __popcll(bal);
    __syncthreads();
    if (need) {
      int before = found + __popcll(bal & ((lane == 0) ? 0ull : (~0ull >> (64 - lane))));
      for (int w = 0; w < wave; ++w) before += wave_cnt_s[w];
      slices_s[before] = static_cast<int16_t>(sl);
    }
    found += wave_cnt_s[0] + wave_cnt_s[1] + wave_cnt_s[2] + wave_cnt_s[3];
    __syncthreads();  // every thread has read the counts before the next round writes them
  }
  const int nslices = found;

  // compute: lane group G = lane/16 holds K rows 8G..8G+7 of a slice for
  // column n0 + lane%16 (transpose reads), and the input pieces of rows
  // 16 mb + lane%16
  const int G = lane >> 4;
  const int pl = lane & 15;
  const int mblocks = (p.M + 15) >> 4;
  f32x4_t acc[4];
#pragma unroll
  for (int mb = 0; mb < 4; ++mb) acc[mb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  // input pieces of slice `i` (zero where the row's support skips it)
  auto load_x = [&](int i, uint4 (&xv)[4]) {
    const int32_t kk = slices_s[i] * SLICE + 8 * G;
    const unsigned long long gm = kk < p.K ? rowmask_s[group_of(S_s, p.q, kk)] : 0ull;
#pragma unroll
    for (int mb = 0; mb < 4; ++mb) {
      const int m = 16 * mb + pl;
      const bool ok = mb < mblocks && m < p.M && ((gm >> m) & 1ull);
      const uint4 xa = *reinterpret_cast<const uint4*>(p.A + (ok ? static_cast<int64_t>(m) * p.K + kk : 0));
      xv[mb] = ok ? xa : make_uint4(0, 0, 0, 0);
    }
  };
  const int pass = p.slots;  // slices held in LDS at once (the launch's LDS room)
  for (int p0 = 0; p0 < nslices; p0 += pass) {
    const int p1 = min(nslices, p0 + pass);
    // stream this wave's slices of the pass into LDS (slot i - p0): lane l
    // carries row l/2, 16 bytes (8 columns) at half l%2.  Rows past K repeat
    // row K-1 and columns past the group repeat its first column (finite
    // values; their products are either multiplied by zero inputs or never
    // stored).
    for (int i = p0 + wave; i < p1; i += 4) {
      int32_t row = slices_s[i] * SLICE + (lane >> 1);
      row = row < p.K ? row : p.K - 1;
      int32_t col = n0 + 8 * (lane & 1);
      col = col < nend ? col : n0;
      const uint16_t* g = p.W + static_cast<int64_t>(row) * p.N + col;
      __builtin_amdgcn_global_load_lds(g, (STARQ_LDS void*)(lds + (i - p0) * 1024), 16, 0, 0);
    }
    __builtin_amdgcn_s_waitcnt(0);
    __builtin_amdgcn_wave_barrier();
    __asm__ volatile("" ::: "memory");
    // the input pieces, prefetched two slices ahead
    uint4 x0[4], x1[4], x2[4];
    if (p0 + wave < p1) load_x(p0 + wave, x0);
    if (p0 + wave + 4 < p1) load_x(p0 + wave + 4, x1);
    for (int i = p0 + wave; i < p1; i += 4) {
      if (i + 8 < p1) load_x(i + 8, x2);
      const char* base = lds + (i - p0) * 1024 + (8 * G + (pl >> 2)) * 32 + (pl & 3) * 8;
      const v4i16_t w0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((STARQ_LDS v4i16_t*)(base));
      const v4i16_t w1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((STARQ_LDS v4i16_t*)(base + 128));
      uint4 wf;
      wf.x = static_cast<uint16_t>(w0[0]) | (static_cast<uint32_t>(static_cast<uint16_t>(w0[1])) << 16);
      wf.y = static_cast<uint16_t>(w0[2]) | (static_cast<uint32_t>(static_cast<uint16_t>(w0[3])) << 16);
      wf.z = static_cast<uint16_t>(w1[0]) | (static_cast<uint32_t>(static_cast<uint16_t>(w1[1])) << 16);
      wf.w = static_cast<uint16_t>(w1[2]) | (static_cast<uint32_t>(static_cast<uint16_t>(w1[3])) << 16);
#pragma unroll
      for (int mb = 0; mb < 4; ++mb) {
        if (mb < mblocks) {
          // D[n][m] += W^T x^T: lane ends with 4 consecutive columns of row m
          acc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, wf),
                                                            __builtin_bit_cast(bf16x8_t, x0[mb]),
                                                            acc[mb], 0, 0, 0);
        }
      }
#pragma unroll
      for (int mb = 0; mb < 4; ++mb) {
        x0[mb] = x1[mb];
        x1[mb] = x2[mb];
      }
    }
    // the wave's slots are free for the next pass once its reads are done
    __builtin_amdgcn_s_waitcnt(0);
    __builtin_amdgcn_wave_barrier();
    __asm__ volatile("" ::: "memory");
  }

  // add the four waves' partial sums in a fixed order
  f32x4_t* red = reinterpret_cast<f32x4_t*>(lds + p.slots * 1024);
#pragma unroll
  for (int mb = 0; mb < 4; ++mb) red[(wave * 4 + mb) * 64 + lane] = acc[mb];
  __syncthreads();
  {
    const int mb = tid >> 6;
    const int l = tid & 63;
    const int m = 16 * mb + (l & 15);
    const int32_t n = n0 + 4 * (l >> 4);
    if (mb < mblocks && m < p.M && n < nend) {
      f32x4_t z = red[(0 * 4 + mb) * 64 + l];
      z += red[(1 * 4 + mb) * 64 + l];
      z += red[(2 * 4 + mb) * 64 + l];
      z += red[(3 * 4 + mb) * 64 + l];
      if (p.bias) {
        const float4 bv = *reinterpret_cast<const float4*>(p.bias + n);
        z[0] += bv.x; z[1] += bv.y; z[2] += bv.z; z[3] += bv.w;
      }
      const int64_t o = static_cast<int64_t>(m) * p.N + n;
      if (p.mode == 0) {
        uint2 w;
        w.x = f32_to_bf16(act_apply(p.act, z[0])) | (static_cast<uint32_t>(f32_to_bf16(act_apply(p.act, z[1]))) << 16);
        w.y = f32_to_bf16(act_apply(p.act, z[2])) | (static_cast<uint32_t>(f32_to_bf16(act_apply(p.act, z[3]))) << 16);
        *reinterpret_cast<uint2*>(p.out_bf16 + o) = w;
      } else {
        float hv[4];
        if (p.residual) {
          if (p.h_init) {
            const uint2 hi = *reinterpret_cast<const uint2*>(p.h_init + o);
            hv[0] = bf16_to_f32(hi.x & 0xffffu); hv[1] = bf16_to_f32(hi.x >> 16);
            hv[2] = bf16_to_f32(hi.y & 0xffffu); hv[3] = bf16_to_f32(hi.y >> 16);
          } else {
            const float4 hp = *reinterpret_cast<const float4*>(p.h_in + o);
            hv[0] = hp.x; hv[1] = hp.y; hv[2] = hp.z; hv[3] = hp.w;
          }
        } else {
          hv[0] = hv[1] = hv[2] = hv[3] = 0.f;
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) hv[e] += z[e];
        if (p.h_out) *reinterpret_cast<float4*>(p.h_out + o) = make_float4(hv[0], hv[1], hv[2], hv[3]);
        if (p.out_bf16) {
          uint2 w;
          w.x = f32_to_bf16(hv[0]) | (static_cast<uint32_t>(f32_to_bf16(hv[1])) << 16);
          w.y = f32_to_bf16(hv[2]) | (static_cast<uint32_t>(f32_to_bf16(hv[3])) << 16);
          *reinterpret_cast<uint2*>(p.out_bf16 + o) = w;
        }
        if (p.Y) {
#pragma unroll
          for (int e = 0; e < 4; ++e) store_out(p.Y, p.ydtype, o + e, hv[e]);
        }
      }
    }
  }
}

}  // namespace

// LDS slots for the slices a workgroup can need: the support of output
// group j over the rows' types reaches at most min(q, M + 1) groups under
// the star and graph laws (B(t, j) within {t, j}), every group under the
// others; a group of s inputs spans at most ceil(s / 32) + 1 slices.  Fewer
// slots let more workgroups share a CU (a single row at q = 32 needs about
// 10 of the 128).
int decode_phase_slots(const DecodePhase& p) {
  const int reach = (p.law == 0 || p.law == 3) ? std::min(p.q, p.M + 1) : p.q;
  int widest = 0;
  for (int g = 0; g < p.q; ++g) widest = std::max(widest, (p.S[g + 1] - p.S[g] + SLICE - 1) / SLICE + 1);
  const int nsl = (p.K + SLICE - 1) / SLICE;
  return std::max(1, std::min({kPassSlices, nsl, reach * widest}));
}

size_t decode_phase_smem(int slots) { return static_cast<size_t>(slots) * 1024 + kRedBytes; }

hipError_t launch_decode_phase(DecodePhase p, hipStream_t stream) {
  static std::atomic<unsigned long long> lds_set{0};
  const hipError_t attr = ensure_lds_limit(reinterpret_cast<const void*>(decode_phase_kernel), lds_set,
                                           static_cast<int>(decode_phase_smem(kPassSlices)));
  if (attr != hipSuccess) return attr;
  p.slots = decode_phase_slots(p);
  const int nt = p.NTp[p.q];
  const int grid = (nt + 31) / 32 * 32;
  hipLaunchKernelGGL(decode_phase_kernel, dim3(grid), dim3(kThreads), decode_phase_smem(p.slots), stream, p);
  return hipGetLastError();
}

}  // namespace starq
