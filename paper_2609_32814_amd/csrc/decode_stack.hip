// The decode stack (§"One-Token Inference": every layer's FFN applies the
// row-typed projection with the token's row type) as one persistent kernel.
//
// Per layer two projections run back to back: up (D -> F, bias, GELU) and
// down (F -> D, bias, residual).  A workgroup owns one 16-column tile of
// each: up tiles cover F with the whole K = D; down tiles cover D with K = F
// cut into ns chunks of kc, so both phases have about the same number of
// equal items and every item streams the same amount of weight.  Within an
// item the compute follows the per-phase decode kernel: only the 32-row
// weight slices that some row's support reaches are copied, inputs of rows
// whose support skips a slice are zero, v_mfma_f32_16x16x32_bf16 over up to
// 64 rows, and the four wavefronts' sums are added in a fixed order.
//
// What the single launch buys: a workgroup copies the weights of its next
// up (down) item into LDS as soon as the current one is consumed, before it
// waits for the other workgroups, so the weight stream runs ahead of the
// layer-to-layer dependencies instead of starting at each kernel boundary.
//
// Cross-workgroup data (H, the next layer's input, the residual, the
// partial sums) is written with agent-coherent stores and read with
// agent-coherent loads (copies into LDS with sc0 sc1), so no cache
// write-back or invalidate is needed; arrival counters are agent-scope
// atomics that only grow (a layer's target is a multiple of the item
// count).  The down chunks of one tile are summed by whichever of its
// workgroups arrives last, in chunk order, so results do not depend on
// timing.  Every wait is bounded: after about half a second of spinning the
// kernel raises the error flag and carries on, so it always terminates.
#include "common.hpp"
#include "kernels.hpp"

namespace starq {

namespace {

constexpr int kThreads = 256;
constexpr int TN = 16;          // output columns per item
constexpr int SLICE = 32;       // K rows per weight slice (1 KB)
constexpr int kMaxSlices = 32;  // per item (K chunk <= 1024)
constexpr int kRedBytes = 4 * 4 * 64 * 16;
constexpr int kSpinLimit = 1 << 18;  // about 0.5 s per wait

typedef short v4i16_t __attribute__((ext_vector_type(4)));
#define STARQ_LDS __attribute__((address_space(3)))

__device__ __attribute__((aligned(256))) uint32_t g_stack_zero[64];

__device__ __forceinline__ void dma16_sys(const void* g, uint32_t lds_addr) {
  // agent-coherent (sc1): reads what other workgroups stored, past this
  // XCD's L2
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off sc1"
               :
               : "v"(g), "s"(lds_addr)
               : "memory", "m0");
}
__device__ __forceinline__ void dma16(const void* g, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(g), "s"(lds_addr)
               : "memory", "m0");
}
__device__ __forceinline__ void wait_vm_all() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));
  asm volatile("" ::: "memory");
}
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(reinterpret_cast<uintptr_t>(p)));
}

__device__ __forceinline__ void st_agent(uint32_t* p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t ld_agent(const uint32_t* p) {
  return __hip_atomic_load(const_cast<uint32_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ bool in_support(int law, int i, int j, int k) {
  return law == 1 || k == i || k == j;
}
__device__ __forceinline__ int group_of(const int32_t* starts, int q, int32_t x) {
  int g = 0;
  while (g + 1 < q && x >= starts[g + 1]) ++g;
  return g;
}

// One projection item: 16 output columns [n0, nend) of output group j, K
// range [k_lo, k_hi) of an input with row stride ldx and weight row stride
// ldw.
struct Item {
  int32_t valid;
  int32_t j, n0, nend, k_lo, k_hi;
};

__device__ __forceinline__ Item up_item(const DecodeStack& p) {
  Item it{};
  const int ct = blockIdx.x;
  it.valid = ct < p.nt_up;
  if (!it.valid) return it;
  int j = 0;
  while (ct >= p.NTu[j + 1]) ++j;
  it.j = j;
  it.n0 = p.SF[j] + (ct - p.NTu[j]) * TN;
  it.nend = p.SF[j + 1];
  it.k_lo = 0;
  it.k_hi = p.D;
  return it;
}

__device__ __forceinline__ Item down_item(const DecodeStack& p) {
  Item it{};
  const int d = blockIdx.x;
  it.valid = d < p.nt_dn * p.ns;
  if (!it.valid) return it;
  const int ct = d / p.ns, s = d % p.ns;
  int j = 0;
  while (ct >= p.NTd[j + 1]) ++j;
  it.j = j;
  it.n0 = p.SD[j] + (ct - p.NTd[j]) * TN;
  it.nend = p.SD[j + 1];
  it.k_lo = s * p.kc;
  it.k_hi = min(p.F, (s + 1) * p.kc);
  return it;
}

__global__ __launch_bounds__(kThreads) void decode_stack_kernel(const DecodeStack p) {
  extern __shared__ __attribute__((aligned(16))) char lds[];
  // per weight slot (0: up item, 1: down item): rows needing each K group,
  // the needed slices
  __shared__ unsigned long long rowmask_s[2][kMaxQGroups];
  __shared__ int16_t slices_s[2][kMaxSlices];
  // rows whose support reaches each 8-wide piece of each needed slice
  __shared__ unsigned long long pmask_s[2][kMaxSlices][4];
  __shared__ int32_t nslices_s[2];
  __shared__ int32_t wave_cnt_s[2];
  __shared__ int32_t flag_s;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int M = p.M;
  const int mblocks = (M + 15) >> 4;
  const int kmax = (max(p.D, p.kc) + 127) & ~127;
  // staging writes whole 1 KB copies, so round the x buffer up to 1 KB
  const int xbytes = max((M * kmax * 2 + 1023) & ~1023, kRedBytes);
  char* xbuf = lds;
  char* slot_base[2] = {lds + xbytes, lds + xbytes + (kmax / SLICE) * 1024};
  int32_t* cnt_up = p.cnt;
  int32_t* cnt_dn = p.cnt + 1;
  int32_t* err = p.cnt + 2;
  int32_t* tile_cnt = p.cnt + 3;
  const void* zero = g_stack_zero;

  const Item iu = up_item(p);
  const Item idn = down_item(p);

  // Which rows need input group g for output group j (one ballot per
  // group by wave 0), then the needed slices of [k_lo, k_hi) in K order,
  // then the copies of those slices of W into the slot.
  auto plan_and_copy = [&](int slot, const Item& it, const int32_t* KS, const uint16_t* W,
                           int32_t ldw) {
    if (wave == 0) {
      const int t = lane < M ? p.types[lane] : -1;
      for (int g = 0; g < p.q; ++g) {
        const unsigned long long m = __ballot(lane < M && in_support(p.law, t, it.j, g));
        if (lane == 0) rowmask_s[slot][g] = m;
      }
    }
    __syncthreads();
    const int nsl = (it.k_hi - it.k_lo + SLICE - 1) / SLICE;  // <= kMaxSlices
    bool need = false;
    if (tid < nsl) {
      for (int piece = 0; piece < SLICE / 8; ++piece) {
        const int32_t k = it.k_lo + tid * SLICE + piece * 8;
        if (k < it.k_hi && rowmask_s[slot][group_of(KS, p.q, k)]) need = true;
      }
    }
    const unsigned long long bal = __ballot(need);
    if (wave == 0 && lane == 0) wave_cnt_s[slot] = __popcll(bal);
    __syncthreads();
    if (need) {
      const int before = __popcll(bal & ((lane == 0) ? 0ull : (~0ull >> (64 - lane))));
      slices_s[slot][before] = static_cast<int16_t>(tid);
    }
    if (tid == 0) nslices_s[slot] = wave_cnt_s[slot];
    __syncthreads();
    const int ns_ = nslices_s[slot];
    if (tid < 4 * ns_) {
      const int32_t k = it.k_lo + slices_s[slot][tid >> 2] * SLICE + 8 * (tid & 3);
      pmask_s[slot][tid >> 2][tid & 3] = k < it.k_hi ? rowmask_s[slot][group_of(KS, p.q, k)] : 0ull;
    }
    // (read by compute after the barrier that precedes it)
    char* sb = slot_base[slot];
    for (int i = wave; i < ns_; i += 4) {
      int32_t row = it.k_lo + slices_s[slot][i] * SLICE + (lane >> 1);
      row = row < it.k_hi ? row : it.k_hi - 1;  // finite filler, its inputs are zero
      int32_t col = it.n0 + 8 * (lane & 1);
      col = col < it.nend ? col : it.n0;
      dma16(W + static_cast<int64_t>(row) * ldw + col, lds_addr(sb + i * 1024));
    }
  };

  // Bounded wait until *c >= target (thread 0 spins, the others wait at the
  // barrier).
  auto wait_for = [&](int32_t* c, int32_t target) {
    if (tid == 0) {
      int spins = 0;
      while (static_cast<int32_t>(ld_agent(reinterpret_cast<uint32_t*>(c))) < target) {
        __builtin_amdgcn_s_sleep(1);
        if (++spins > kSpinLimit) {
          st_agent(reinterpret_cast<uint32_t*>(err), 1u);
          break;
        }
      }
    }
    __syncthreads();
  };

  // Stage the item's inputs (rows < M, K range rounded up to 128) into the
  // swizzled x buffer: chunk c of row m at chunk c ^ (m & 15), so the 16
  // rows of an MFMA operand read hit distinct banks.  Inputs past k_hi or
  // past M are zero.
  auto stage_x = [&](const Item& it, const uint16_t* src, int32_t ldx) {
    const int kx = (it.k_hi - it.k_lo + 127) & ~127;
    const int cpr = kx / 8;  // 16-byte chunks per row, a multiple of 16
    const int total = M * cpr;
    for (int f0 = wave * 64; f0 < total; f0 += 256) {
      const int f = f0 + lane;
      const int m = f / cpr;
      const int pc = f - m * cpr;
      const int c = pc ^ (m & 15);
      const int32_t k = it.k_lo + 8 * c;
      const bool ok = f < total && k < it.k_hi;
      const void* g = ok ? static_cast<const void*>(src + static_cast<int64_t>(m) * ldx + k) : zero;
      dma16_sys(g, lds_addr(xbuf + f0 * 16));
    }
  };

  // acc over the item's slices; lane group G = lane / 16 holds K rows
  // 8G..8G+7 of a slice for column n0 + lane % 16, and rows 16 mb + lane % 16
  auto compute = [&](int slot, const Item& it, f32x4_t (&acc)[4]) {
    const int G = lane >> 4;
    const int pl = lane & 15;
    const int kx = (it.k_hi - it.k_lo + 127) & ~127;
    const int ns_ = nslices_s[slot];
    const char* sb = slot_base[slot];
#pragma unroll
    for (int mb = 0; mb < 4; ++mb) acc[mb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    // operands of slice i: the weight fragment and the masked input pieces
    auto load = [&](int i, uint4& wf, uint4 (&xv)[4]) {
      const char* base = sb + i * 1024 + (8 * G + (pl >> 2)) * 32 + (pl & 3) * 8;
      const v4i16_t w0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((STARQ_LDS v4i16_t*)(base));
      const v4i16_t w1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((STARQ_LDS v4i16_t*)(base + 128));
      wf.x = static_cast<uint16_t>(w0[0]) | (static_cast<uint32_t>(static_cast<uint16_t>(w0[1])) << 16);
      wf.y = static_cast<uint16_t>(w0[2]) | (static_cast<uint32_t>(static_cast<uint16_t>(w0[3])) << 16);
      wf.z = static_cast<uint16_t>(w1[0]) | (static_cast<uint32_t>(static_cast<uint16_t>(w1[1])) << 16);
      wf.w = static_cast<uint16_t>(w1[2]) | (static_cast<uint32_t>(static_cast<uint16_t>(w1[3])) << 16);
      const int32_t krel = slices_s[slot][i] * SLICE + 8 * G;
      const unsigned long long gm = pmask_s[slot][i][G];
#pragma unroll
      for (int mb = 0; mb < 4; ++mb) {
        if (mb < mblocks) {
          const int m = 16 * mb + pl;
          const int mr = min(m, M - 1);  // rows past M read row M - 1, then zero
          const int c = (krel >> 3) ^ (mr & 15);
          xv[mb] = *reinterpret_cast<const uint4*>(xbuf + (mr * kx + 8 * c) * 2);
          if (!(m < M && ((gm >> m) & 1ull))) xv[mb] = make_uint4(0, 0, 0, 0);
        }
      }
    };
    auto mfma = [&](const uint4& wf, const uint4 (&xv)[4]) {
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
        if (mb < mblocks)
          // D[n][m] += W^T x^T: the lane ends with 4 consecutive columns of row m
          acc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, wf),
                                                            __builtin_bit_cast(bf16x8_t, xv[mb]),
                                                            acc[mb], 0, 0, 0);
    };
    // two slices per round: both slices' LDS reads are in flight together
    for (int i0 = wave; i0 < ns_; i0 += 8) {
      uint4 wf0, wf1, xv0[4], xv1[4];
      load(i0, wf0, xv0);
      const bool two = i0 + 4 < ns_;
      if (two) load(i0 + 4, wf1, xv1);
      mfma(wf0, xv0);
      if (two) mfma(wf1, xv1);
    }
  };

  // Fixed-order sum of the four waves' partials (through LDS, reusing the
  // x buffer); thread tid then owns rows 16 mb + l % 16, columns
  // n0 + 4 (l / 16) .. + 3 with mb = tid / 64, l = tid % 64.
  auto reduce = [&](f32x4_t (&acc)[4], f32x4_t& z) {
    __syncthreads();  // every wave is done with the x buffer
    f32x4_t* red = reinterpret_cast<f32x4_t*>(xbuf);
#pragma unroll
    for (int mb = 0; mb < 4; ++mb) red[(wave * 4 + mb) * 64 + lane] = acc[mb];
    __syncthreads();
    const int mb = tid >> 6;
    z = red[(0 * 4 + mb) * 64 + lane];
    z += red[(1 * 4 + mb) * 64 + lane];
    z += red[(2 * 4 + mb) * 64 + lane];
    z += red[(3 * 4 + mb) * 64 + lane];
  };

  const int my_m = 16 * (tid >> 6) + (lane & 15);
  const int my_dn = 4 * (lane >> 4);

  // prologue: weights of layer 0's items
  if (iu.valid) plan_and_copy(0, iu, p.SD, p.Wu[0], p.F);
  if (idn.valid) plan_and_copy(1, idn, p.SF, p.Wd[0], p.D);

  for (int l = 0; l < p.L; ++l) {
    // ---------------- up projection: H = act(x W_up + b_up) ----------------
    if (l > 0) wait_for(cnt_dn, p.nt_dn * l);
    if (iu.valid) {
      const uint16_t* xin = (l == 0) ? p.X : p.hb + static_cast<int64_t>(l & 1) * M * p.D;
      stage_x(iu, xin, p.D);
      wait_vm_all();
      __syncthreads();
      f32x4_t acc[4], z;
      compute(0, iu, acc);
      reduce(acc, z);
      const int32_t n = iu.n0 + my_dn;
      if (my_m < M && n < iu.nend) {
        const float* b = p.bu[l];
        float v[4] = {z[0], z[1], z[2], z[3]};
        if (b) {
          const float4 bv = *reinterpret_cast<const float4*>(b + n);
          v[0] += bv.x; v[1] += bv.y; v[2] += bv.z; v[3] += bv.w;
        }
        uint32_t* dst = reinterpret_cast<uint32_t*>(p.H + static_cast<int64_t>(my_m) * p.F + n);
        st_agent(dst, f32_to_bf16(act_fwd(p.act, v[0])) |
                          (static_cast<uint32_t>(f32_to_bf16(act_fwd(p.act, v[1]))) << 16));
        st_agent(dst + 1, f32_to_bf16(act_fwd(p.act, v[2])) |
                              (static_cast<uint32_t>(f32_to_bf16(act_fwd(p.act, v[3]))) << 16));
      }
      wait_vm_all();  // the stores have reached the coherent level
      __syncthreads();
      if (tid == 0) __hip_atomic_fetch_add(cnt_up, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      // slot 0 is free (every wave passed the barriers above): the next
      // layer's up weights stream in while this workgroup waits
      if (l + 1 < p.L) plan_and_copy(0, iu, p.SD, p.Wu[l + 1], p.F);
    }

    // ---------------- down projection: h += H W_down + b_down ----------------
    wait_for(cnt_up, p.nt_up * (l + 1));
    if (idn.valid) {
      const int ct = blockIdx.x / p.ns, s = blockIdx.x % p.ns;
      stage_x(idn, p.H, p.F);
      wait_vm_all();
      __syncthreads();
      f32x4_t acc[4], z;
      compute(1, idn, acc);
      reduce(acc, z);
      const int32_t n = idn.n0 + my_dn;
      const bool mine = my_m < M && n < idn.nend;
      if (mine) {
        uint32_t* dst = reinterpret_cast<uint32_t*>(p.part + (static_cast<int64_t>(s) * M + my_m) * p.D + n);
#pragma unroll
        for (int e = 0; e < 4; ++e) st_agent(dst + e, __float_as_uint(z[e]));
      }
      wait_vm_all();
      __syncthreads();
      if (tid == 0) {
        const int old = __hip_atomic_fetch_add(tile_cnt + ct, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        flag_s = (old == p.ns * (l + 1) - 1);
      }
      __syncthreads();
      if (flag_s) {
        // last chunk of this tile to arrive: sum the chunks in order
        if (mine) {
          float v[4] = {0.f, 0.f, 0.f, 0.f};
          for (int c = 0; c < p.ns; ++c) {
            const uint32_t* src = reinterpret_cast<const uint32_t*>(
                p.part + (static_cast<int64_t>(c) * M + my_m) * p.D + n);
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] += __uint_as_float(ld_agent(src + e));
          }
          const float* b = p.bd[l];
          if (b) {
            const float4 bv = *reinterpret_cast<const float4*>(b + n);
            v[0] += bv.x; v[1] += bv.y; v[2] += bv.z; v[3] += bv.w;
          }
          const int64_t o = static_cast<int64_t>(my_m) * p.D + n;
          if (p.residual) {
            if (l == 0) {
              const uint2 xi = *reinterpret_cast<const uint2*>(p.X + o);
              v[0] += bf16_to_f32(xi.x & 0xffffu); v[1] += bf16_to_f32(xi.x >> 16);
              v[2] += bf16_to_f32(xi.y & 0xffffu); v[3] += bf16_to_f32(xi.y >> 16);
            } else {
              const uint32_t* hs = reinterpret_cast<const uint32_t*>(p.h + o);
#pragma unroll
              for (int e = 0; e < 4; ++e) v[e] += __uint_as_float(ld_agent(hs + e));
            }
          }
          if (l + 1 < p.L) {
            uint32_t* hd = reinterpret_cast<uint32_t*>(p.h + o);
#pragma unroll
            for (int e = 0; e < 4; ++e) st_agent(hd + e, __float_as_uint(v[e]));
            uint32_t* xd = reinterpret_cast<uint32_t*>(p.hb + static_cast<int64_t>((l + 1) & 1) * M * p.D + o);
            st_agent(xd, f32_to_bf16(v[0]) | (static_cast<uint32_t>(f32_to_bf16(v[1])) << 16));
            st_agent(xd + 1, f32_to_bf16(v[2]) | (static_cast<uint32_t>(f32_to_bf16(v[3])) << 16));
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) store_out(p.Y, p.ydtype, o + e, v[e]);
          }
        }
        wait_vm_all();
        __syncthreads();
        if (tid == 0) __hip_atomic_fetch_add(cnt_dn, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      if (l + 1 < p.L) plan_and_copy(1, idn, p.SF, p.Wd[l + 1], p.D);
    }
  }
  wait_vm_all();
}

}  // namespace

size_t decode_stack_smem(int M, int kmax) {
  if (M < 1 || M > kDecodeMaxRows || kmax < SLICE || kmax > kMaxSlices * SLICE) return 0;
  kmax = (kmax + 127) & ~127;
  const size_t xbytes = std::max<size_t>((static_cast<size_t>(M) * kmax * 2 + 1023) & ~size_t(1023), kRedBytes);
  const size_t total = xbytes + 2 * static_cast<size_t>(kmax / SLICE) * 1024;
  return total <= 150 * 1024 ? total : 0;
}

hipError_t launch_decode_stack(const DecodeStack& p, int grid, hipStream_t stream) {
  const size_t smem = decode_stack_smem(p.M, std::max(p.D, p.kc));
  if (smem == 0) return hipErrorInvalidValue;
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(decode_stack_kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
      150 * 1024);
  if (attr != hipSuccess) return attr;
  DecodeStack arg = p;
  void* args[] = {&arg};
  return hipLaunchCooperativeKernel(reinterpret_cast<const void*>(decode_stack_kernel), dim3(grid),
                                    dim3(kThreads), args, static_cast<unsigned>(smem), stream);
}

}  // namespace starq
