// Grouped, row-typed GEMM for bf16 operands with an asynchronous LDS
// pipeline: the forward projection and its activation gradient.
//
// The tile decomposition, schedule and epilogue follow the register-staged
// kernel (tiles of 256 rows x 128 columns of C, 4 wavefronts of 128 x 64,
// swapped-operand v_mfma_f32_32x32x16_bf16, two passes of tiles, XCD
// chunks); what differs is how operands reach LDS.  Every operand byte goes
// from global memory straight into LDS with global_load_lds_dwordx4 (16
// bytes per lane, 1 KB per wavefront instruction) into a ring of three 48 KB
// stages, so two K steps are in flight while a third is multiplied and no
// staging registers are spent.  A K step waits only for its own stage
// (vmcnt) and one workgroup barrier.  The load side walks the tile sequence
// two stages ahead of the compute side, across tile boundaries.
//
// Everything else a tile needs from memory also arrives by direct copies
// counted in the same stage: the gathered row indices of the next tile and
// the bias of the current one.  A plain load whose value is used would make
// the compiler wait for every copy in flight (it does not see the copies).
// Lanes whose element lies outside an operand (rows past a type's count, K
// or columns past a group's end) copy from a page of zeros.
//
// LDS layouts, per stage:
//  * K-contiguous rows (X and dY rows, and W read as W^T): 128 bytes
//    (64 bf16) per row, the 16-byte chunk c of row r stored at chunk
//    c ^ (r & 7).  Eight lanes of a copy fill one row (the global side reads
//    the row's 128 contiguous bytes, permuted across lanes); a 32-row MFMA
//    operand read touches 8 distinct chunk slots per 8 rows.
//  * N-contiguous rows (W in the forward product): 64 K rows of 128 columns
//    (256 bytes), chunk c of K row k stored at chunk c ^ 2 (k & 3).  The
//    operand read uses ds_read_b64_tr_b16: in each 16-lane group, lanes
//    4r + q point at columns 4q..4q+3 of K row r and lane i receives column i
//    of those 4 rows, so two reads give a lane 8 consecutive K values of one
//    column, which is the MFMA operand layout.
#include <algorithm>

#include "gemm_common.hpp"

namespace starq {

namespace {

using namespace gemm;

constexpr int BN = 128;
constexpr int BK = 32;
constexpr int STAGES = 3;
constexpr int A_BYTES = BM * BK * 2;            // 256 rows x 32 bf16: 16 KB
constexpr int B_BYTES = BN * BK * 2;            // 128 columns x 32 bf16: 8 KB
constexpr int STAGE_BYTES = A_BYTES + B_BYTES;  // 24 KB
constexpr int SMEM = STAGES * STAGE_BYTES;      // 72 KB: two workgroups per CU
constexpr int DMA_A = A_BYTES / 1024 / 4;       // A copies per wave per stage (4)
constexpr int DMA_B = B_BYTES / 1024 / 4;       // B copies per wave per stage (2)
constexpr int kRowBufs = 4;                     // row-index / bias buffers

// copies per wave per stage: A, B, next tile's row indices, (bias)
template <int MODE>
constexpr int stage_ops() {
  return DMA_A + DMA_B + (MODE == kModeFwd ? 2 : 1);
}

typedef short v4i16_t __attribute__((ext_vector_type(4)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
#define STARQ_LDS __attribute__((address_space(3)))

// 256 zero bytes: the source of every copy whose element lies outside an
// operand.
__device__ __attribute__((aligned(256))) uint32_t g_zero_page[64];

// 16 (dma16) or 4 (dma4) bytes per lane from global memory into LDS at
// lds_addr + 16 * lane (4 * lane).  Issued as assembly so that the
// compiler's wait-count bookkeeping, which would otherwise drain every copy
// in flight before any LDS read, stays out of the pipeline; the waits below
// are explicit.
__device__ __forceinline__ void dma16(const void* g, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(g), "s"(lds_addr)
               : "memory", "m0");
}
__device__ __forceinline__ void dma4(const void* g, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dword %0, off"
               :
               : "v"(g), "s"(lds_addr)
               : "memory", "m0");
}

// Wait until at most N vector-memory operations of this wave are in flight.
// Loads complete in order, so this covers every copy issued before the last
// N; stores issued in between only make it wait longer.
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
  asm volatile("" ::: "memory");
}

__device__ __forceinline__ void block_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return __builtin_amdgcn_readfirstlane(
      static_cast<uint32_t>(reinterpret_cast<uintptr_t>(p)));
}

// byte offset of 16-byte chunk c (0..3) of row r in a K-contiguous tile of
// 64-byte rows; rows r and r ^ 1 share a 128-byte bank line, so the chunk
// is rotated by (r >> 1) & 3 and 8 consecutive rows hit 8 distinct 16-byte
// bank groups
__device__ __forceinline__ int krow_off(int r, int c) { return r * 64 + ((c ^ ((r >> 1) & 3)) << 4); }
// byte offset of column chunk c of K row k in an N-contiguous 128-column tile
__device__ __forceinline__ int kcol_off(int k, int c) { return k * 256 + ((c ^ (2 * (k & 3))) << 4); }

__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a, b}, bf16x2_t));
}

__device__ __forceinline__ void store4_out(void* base, int dtype, int64_t idx, const float (&v)[4]) {
  if (dtype == 0) {
    *reinterpret_cast<float4*>(static_cast<float*>(base) + idx) = make_float4(v[0], v[1], v[2], v[3]);
  } else {
    uint2 w;
    w.x = pack_bf16(v[0], v[1]);
    w.y = pack_bf16(v[2], v[3]);
    *reinterpret_cast<uint2*>(static_cast<uint16_t*>(base) + idx) = w;
  }
}

// Workgroups per CU: two, so that one's epilogue and waits overlap the
// other's MFMA work; one for the activation gradient with Z_prev, whose
// epilogue needs more than the 256 registers a lane has at two per CU.
template <int MODE, int ACT>
constexpr int occupancy() {
  return (MODE == kModeBwdData && ACT != kActNone) ? 1 : 2;
}

template <int MODE, int LAW, int ACT>
__global__ __launch_bounds__(THREADS, (occupancy<MODE, ACT>())) void star_gemm_async_kernel(const GemmParams p) {
  constexpr int OPS = stage_ops<MODE>();
  extern __shared__ __attribute__((aligned(16))) char smem[];
  __shared__ int32_t units_s[kMaxQGroups];
  __shared__ int32_t offs_s[kMaxQGroups + 1];
  __shared__ int32_t pfx_s[2][kMaxQGroups + 1];
  __shared__ __attribute__((aligned(16))) int32_t rows_s[kRowBufs][BM];
  __shared__ __attribute__((aligned(16))) float bias_s[kRowBufs][BN];
  __shared__ __attribute__((aligned(16))) float junk_s[64];

  const uint16_t* __restrict__ Ag = static_cast<const uint16_t*>(p.A);
  const uint16_t* __restrict__ Bg = static_cast<const uint16_t*>(p.B);
  const void* zero = g_zero_page;
  const int q = p.q;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int lr = lane & 31, lh = lane >> 5;

  for (int i = threadIdx.x; i <= q; i += THREADS) offs_s[i] = p.offsets[i];
  __syncthreads();
  for (int i = threadIdx.x; i < q; i += THREADS) units_s[i] = (offs_s[i + 1] - offs_s[i] + BM - 1) / BM;
  __syncthreads();
  if (threadIdx.x < 2) {
    const int sel = sel_for(MODE, LAW, threadIdx.x);
    int32_t run = 0;
    for (int i = 0; i < q; ++i) {
      pfx_s[threadIdx.x][i] = run;
      run += units_s[i] * ncols_sel(p, sel, i);
    }
    pfx_s[threadIdx.x][q] = run;
  }
  __syncthreads();

  // ---- tile iterators (the compute side and the load side walk one list) ----
  const int xcd = blockIdx.x & 7;
  const int slot_stride = gridDim.x >> 3;
  struct Iter {
    int pass;
    int32_t slot;
  };
  auto advance = [&](Iter& it, Tile& t) -> bool {
    while (it.pass < 2) {
      const int32_t total = pfx_s[it.pass][q];
      const int32_t chunk = (total + 7) >> 3;
      const int32_t logical = xcd * chunk + it.slot;
      if (it.slot >= chunk || logical >= total) {
        ++it.pass;
        it.slot = blockIdx.x >> 3;
        continue;
      }
      it.slot += slot_stride;
      int cls = 0;
      while (logical >= pfx_s[it.pass][cls + 1]) ++cls;
      t = make_tile<MODE, LAW, BN, BK>(p, sel_for(MODE, LAW, it.pass), cls,
                                       logical - pfx_s[it.pass][cls], units_s[cls], offs_s);
      return true;
    }
    return false;
  };

  Iter cit{0, static_cast<int32_t>(blockIdx.x >> 3)};
  Tile ct;
  if (!advance(cit, ct)) return;

  // ---- load side: tile lt (sequence number lseq, step ls), next tile ln ----
  Iter lit = cit;
  Tile lt = ct, ln;
  int32_t lseq = 0, ls = 0;
  bool lvalid = true;
  bool rows_from_lds = false;  // rl must be refilled from rows_s
  int32_t rl[DMA_A];  // gathered row of A copy j: tile row 16 (wave + 4 j) + lane / 4
#pragma unroll
  for (int j = 0; j < DMA_A; ++j) {
    const int row = 16 * (wave + 4 * j) + (lane >> 2);
    rl[j] = row < lt.nrows ? p.perm[lt.pos0 + row] : -1;
  }
  bool has_ln = advance(lit, ln);

  auto issue_stage = [&](int slot) {
    char* As = smem + slot * STAGE_BYTES;
    char* Bs = As + A_BYTES;
    if (!lvalid) {
      // nothing left to load: keep the per-stage number of copies uniform
#pragma unroll
      for (int j = 0; j < OPS; ++j) dma16(zero, lds_addr(As + wave * 1024));
      return;
    }
    if (rows_from_lds) {
#pragma unroll
      for (int j = 0; j < DMA_A; ++j) {
        const int row = 16 * (wave + 4 * j) + (lane >> 2);
        rl[j] = row < lt.nrows ? rows_s[lseq & (kRowBufs - 1)][row] : -1;
      }
      rows_from_lds = false;
    }
    int32_t k0, kend;
    if (ls < lt.n0) {
      k0 = lt.seg0_lo + ls * BK;
      kend = lt.seg0_hi;
    } else {
      k0 = lt.seg1_lo + (ls - lt.n0) * BK;
      kend = lt.seg1_hi;
    }
    const int64_t lda = (MODE == kModeFwd) ? p.K : p.N;
    // A: gathered K-contiguous rows, 16 rows per copy
#pragma unroll
    for (int j = 0; j < DMA_A; ++j) {
      const int ii = wave + 4 * j;
      const int row = 16 * ii + (lane >> 2);
      const int c = (lane & 3) ^ ((row >> 1) & 3);
      const int32_t k = k0 + 8 * c;
      const bool ok = rl[j] >= 0 && k < kend;
      const void* g = ok ? static_cast<const void*>(Ag + static_cast<int64_t>(rl[j]) * lda + k) : zero;
      dma16(g, lds_addr(As + ii * 1024));
    }
    if constexpr (MODE == kModeFwd) {
      // B = W[k][n], N-contiguous: 4 K rows per copy
#pragma unroll
      for (int j = 0; j < DMA_B; ++j) {
        const int ii = wave + 4 * j;
        const int kr = 4 * ii + (lane >> 4);
        const int c = (lane & 15) ^ (2 * (kr & 3));
        const int32_t k = k0 + kr;
        const int32_t col = lt.cstart + 8 * c;
        const bool ok = k < kend && col < lt.cend;
        const void* g = ok ? static_cast<const void*>(Bg + static_cast<int64_t>(k) * p.N + col) : zero;
        dma16(g, lds_addr(Bs + ii * 1024));
      }
    } else {
      // B = rows kk of W read as W^T, K-contiguous (along n): 16 rows per copy
#pragma unroll
      for (int j = 0; j < DMA_B; ++j) {
        const int ii = wave + 4 * j;
        const int row = 16 * ii + (lane >> 2);
        const int c = (lane & 3) ^ ((row >> 1) & 3);
        const int32_t kk = lt.cstart + row;
        const int32_t n = k0 + 8 * c;
        const bool ok = kk < lt.cend && n < kend;
        const void* g = ok ? static_cast<const void*>(Bg + static_cast<int64_t>(kk) * p.N + n) : zero;
        dma16(g, lds_addr(Bs + ii * 1024));
      }
    }
    {
      // row indices of the next tile (the same copy at every step of lt)
      const int r = 64 * wave + lane;
      const void* g = (has_ln && r < ln.nrows) ? static_cast<const void*>(p.perm + ln.pos0 + r) : zero;
      dma4(g, lds_addr(&rows_s[(lseq + 1) & (kRowBufs - 1)][64 * wave]));
    }
    if constexpr (MODE == kModeFwd) {
      // bias of this tile's columns: waves 0 and 1 copy 64 each
      if (wave < 2) {
        const int32_t col = lt.cstart + 64 * wave + lane;
        const void* g = (p.bias && col < lt.cend) ? static_cast<const void*>(p.bias + col) : zero;
        dma4(g, lds_addr(&bias_s[lseq & (kRowBufs - 1)][64 * wave]));
      } else {
        dma4(zero, lds_addr(junk_s));
      }
    }
    if (++ls == lt.nsteps) {
      if (has_ln) {
        // Every tile has three or more K steps of 32 (the host sends
        // groups of 64 or fewer columns to the register-staged kernel), so
        // the first copy of ln's rows was issued at least two stages back
        // and has landed by the next issue.
        rows_from_lds = true;
        lt = ln;
        ++lseq;
        ls = 0;
        has_ln = advance(lit, ln);
      } else {
        lvalid = false;
      }
    }
  };

  // fragments of one 16-wide K slice
  auto read_frags = [&](const char* As, const char* Bs, int rs, uint4 (&fa)[4], uint4 (&fb)[2]) {
    const int kp = 2 * rs + lh;
#pragma unroll
    for (int mi = 0; mi < 4; ++mi) {
      const int row = wm * 128 + mi * 32 + lr;
      fa[mi] = *reinterpret_cast<const uint4*>(As + krow_off(row, kp));
    }
    if constexpr (MODE == kModeFwd) {
      const int gq = lane >> 4, pp = lane & 15;
      const int k = 16 * rs + 8 * (gq >> 1) + (pp >> 2);
#pragma unroll
      for (int ni = 0; ni < 2; ++ni) {
        const int col = wn * 64 + ni * 32 + 16 * (gq & 1) + 4 * (pp & 3);
        const char* a0 = Bs + kcol_off(k, col >> 3) + ((col >> 2) & 1) * 8;
        const v4i16_t w0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((STARQ_LDS v4i16_t*)(a0));
        const v4i16_t w1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((STARQ_LDS v4i16_t*)(a0 + 4 * 256));
        fb[ni].x = static_cast<uint16_t>(w0[0]) | (static_cast<uint32_t>(static_cast<uint16_t>(w0[1])) << 16);
        fb[ni].y = static_cast<uint16_t>(w0[2]) | (static_cast<uint32_t>(static_cast<uint16_t>(w0[3])) << 16);
        fb[ni].z = static_cast<uint16_t>(w1[0]) | (static_cast<uint32_t>(static_cast<uint16_t>(w1[1])) << 16);
        fb[ni].w = static_cast<uint16_t>(w1[2]) | (static_cast<uint32_t>(static_cast<uint16_t>(w1[3])) << 16);
      }
    } else {
#pragma unroll
      for (int ni = 0; ni < 2; ++ni) {
        const int row = wn * 64 + ni * 32 + lr;
        fb[ni] = *reinterpret_cast<const uint4*>(Bs + krow_off(row, kp));
      }
    }
  };

  f32x16_t acc[4][2];
#pragma unroll
  for (int mi = 0; mi < 4; ++mi)
#pragma unroll
    for (int ni = 0; ni < 2; ++ni)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[mi][ni][e] = 0.f;

  // prologue: the first tile's rows for its epilogue, then stages 0 and 1
  {
    const int r = 64 * wave + lane;
    dma4(r < ct.nrows ? static_cast<const void*>(p.perm + ct.pos0 + r) : zero,
         lds_addr(&rows_s[0][64 * wave]));
  }
#pragma unroll
  for (int i = 0; i < STAGES - 1; ++i) issue_stage(i);

  int32_t cseq = 0, cs = 0;
  int slot = 0;
  while (true) {
    wait_vm<OPS>();   // this wave's copies for stage `slot` have landed
    block_barrier();  // and everyone's; the slot computed last step is free
    issue_stage(slot == 0 ? STAGES - 1 : slot - 1);
    {
      const char* As = smem + slot * STAGE_BYTES;
      const char* Bs = As + A_BYTES;
      uint4 fa[2][4], fb[2][2];
      read_frags(As, Bs, 0, fa[0], fb[0]);
      read_frags(As, Bs, 1, fa[1], fb[1]);
#pragma unroll
      for (int rs = 0; rs < 2; ++rs) {
#pragma unroll
        for (int mi = 0; mi < 4; ++mi)
#pragma unroll
          for (int ni = 0; ni < 2; ++ni) mma(acc[mi][ni], fb[rs][ni], fa[rs][mi], uint16_t());
      }
      constexpr int kReads = 4 + (MODE == kModeFwd ? 4 : 2);
      __builtin_amdgcn_sched_group_barrier(0x100, kReads, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, kReads, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 12, 0);
    }
    slot = (slot + 1 == STAGES) ? 0 : slot + 1;
    if (++cs < ct.nsteps) continue;

    // ---- epilogue of tile ct ----
    // The arithmetic runs over all 128 accumulators of the lane without
    // control flow (so independent values interleave); only the memory
    // accesses are predicated on the row and column being inside the tile.
    {
      const int buf = cseq & (kRowBufs - 1);
      const int64_t ldc = (MODE == kModeFwd) ? p.N : p.K;
      bool rv[4], cv[2][4];
      int64_t rbase[4];
#pragma unroll
      for (int mi = 0; mi < 4; ++mi) {
        const int row = wm * 128 + mi * 32 + lr;
        rv[mi] = row < ct.nrows;
        rbase[mi] = static_cast<int64_t>(rv[mi] ? rows_s[buf][row] : 0) * ldc + ct.cstart;
      }
#pragma unroll
      for (int ni = 0; ni < 2; ++ni)
#pragma unroll
        for (int a = 0; a < 4; ++a) cv[ni][a] = ct.cstart + wn * 64 + ni * 32 + 8 * a + 4 * lh < ct.cend;
      auto lcol = [&](int ni, int a) { return wn * 64 + ni * 32 + 8 * a + 4 * lh; };
      if constexpr (MODE == kModeFwd) {
#pragma unroll
        for (int ni = 0; ni < 2; ++ni)
#pragma unroll
          for (int a = 0; a < 4; ++a) {
            const float4 bv = *reinterpret_cast<const float4*>(&bias_s[buf][lcol(ni, a)]);
#pragma unroll
            for (int mi = 0; mi < 4; ++mi) {
              acc[mi][ni][4 * a + 0] += bv.x;
              acc[mi][ni][4 * a + 1] += bv.y;
              acc[mi][ni][4 * a + 2] += bv.z;
              acc[mi][ni][4 * a + 3] += bv.w;
            }
          }
        if (p.Z) {
#pragma unroll
          for (int mi = 0; mi < 4; ++mi)
#pragma unroll
            for (int ni = 0; ni < 2; ++ni)
#pragma unroll
              for (int a = 0; a < 4; ++a)
                if (rv[mi] && cv[ni][a]) {
                  const float v[4] = {acc[mi][ni][4 * a], acc[mi][ni][4 * a + 1],
                                      acc[mi][ni][4 * a + 2], acc[mi][ni][4 * a + 3]};
                  store4_out(p.Z, p.ydtype, rbase[mi] + lcol(ni, a), v);
                }
        }
        if constexpr (ACT != kActNone) {
#pragma unroll
          for (int mi = 0; mi < 4; ++mi)
#pragma unroll
            for (int ni = 0; ni < 2; ++ni)
#pragma unroll
              for (int e = 0; e < 16; ++e) acc[mi][ni][e] = act_apply(ACT, acc[mi][ni][e]);
        }
      } else if constexpr (ACT != kActNone) {
        // activation gradient: dX *= act'(Z_prev) at the same positions,
        // one 32 x 32 block at a time (the fence keeps the compiler from
        // hoisting every Z_prev load, which would not fit in registers)
#pragma unroll
        for (int mi = 0; mi < 4; ++mi)
#pragma unroll
          for (int ni = 0; ni < 2; ++ni) {
#pragma unroll
            for (int a = 0; a < 4; ++a) {
              float z[4] = {0.f, 0.f, 0.f, 0.f};
              if (rv[mi] && cv[ni][a]) load4(p.Zprev, 1, rbase[mi] + lcol(ni, a), z);
#pragma unroll
              for (int j = 0; j < 4; ++j) acc[mi][ni][4 * a + j] *= act_deriv(ACT, z[j]);
            }
            asm volatile("" ::: "memory");
          }
      }
#pragma unroll
      for (int mi = 0; mi < 4; ++mi)
#pragma unroll
        for (int ni = 0; ni < 2; ++ni)
#pragma unroll
          for (int a = 0; a < 4; ++a)
            if (rv[mi] && cv[ni][a]) {
              const float v[4] = {acc[mi][ni][4 * a], acc[mi][ni][4 * a + 1],
                                  acc[mi][ni][4 * a + 2], acc[mi][ni][4 * a + 3]};
              store4_out(p.Y, p.ydtype, rbase[mi] + lcol(ni, a), v);
            }
    }
    if (!advance(cit, ct)) break;
    ++cseq;
    cs = 0;
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
      for (int ni = 0; ni < 2; ++ni)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[mi][ni][e] = 0.f;
  }
  // every copy into LDS lands before the workgroup ends
  wait_vm<0>();
}

template <int MODE, int LAW, int ACT>
hipError_t launch_one(const GemmParams& p, int64_t upper, int cus, hipStream_t stream) {
  auto kern = star_gemm_async_kernel<MODE, LAW, ACT>;
  static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                                     hipFuncAttributeMaxDynamicSharedMemorySize, SMEM);
  if (attr != hipSuccess) return attr;
  // persistent grid: at most `occupancy` workgroups per CU, a multiple of 8
  // so that every XCD gets the same number
  int64_t grid = std::min<int64_t>(std::max<int64_t>(upper, 1),
                                   static_cast<int64_t>(cus) * occupancy<MODE, ACT>());
  grid = (grid + 7) / 8 * 8;
  hipLaunchKernelGGL(kern, dim3(static_cast<unsigned>(grid)), dim3(THREADS), SMEM, stream, p);
  return hipGetLastError();
}

template <int MODE, int LAW>
hipError_t launch_act(const GemmParams& p, int64_t upper, int cus, hipStream_t stream) {
  switch (p.act) {
    case kActGelu: return launch_one<MODE, LAW, kActGelu>(p, upper, cus, stream);
    case kActGeluTanh: return launch_one<MODE, LAW, kActGeluTanh>(p, upper, cus, stream);
    default: return launch_one<MODE, LAW, kActNone>(p, upper, cus, stream);
  }
}

template <int MODE>
hipError_t launch_async(const GemmParams& p, int64_t upper, int cus, hipStream_t stream) {
  return p.law == 1 ? launch_act<MODE, 1>(p, upper, cus, stream)
                    : launch_act<MODE, 0>(p, upper, cus, stream);
}

}  // namespace

hipError_t launch_gemm_async(int mode, const GemmParams& p, int64_t upper_tiles, int cus,
                             hipStream_t stream) {
  if (mode == kModeFwd) return launch_async<kModeFwd>(p, upper_tiles, cus, stream);
  return launch_async<kModeBwdData>(p, upper_tiles, cus, stream);
}

}  // namespace starq
