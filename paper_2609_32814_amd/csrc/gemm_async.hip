// Grouped, row-typed GEMM for bf16 operands with an asynchronous LDS
// pipeline: the forward projection, its activation gradient and its weight
// gradient.
//
// Tiles of C are 256 rows (of one type class) x 256 columns (of one output
// group), computed by one workgroup of 8 wavefronts (2 x 4, 128 x 64 each,
// swapped-operand v_mfma_f32_32x32x16_bf16 so a lane ends with 4 consecutive
// output columns).  Two passes of tiles (two-segment contractions first),
// dealt out per XCD as one list (the second pass in tiles of 128 rows when
// whole tiles would leave the load uneven); the epilogue follows the
// register-staged kernel.  Weight gradient: C = X^T dY over the type-sorted positions of the
// rows whose support pairs the tile's groups, rows read in place through
// perm (the rows of each stage's 64 positions are copied into LDS one stage
// ahead), split along the positions into deterministic partials.
//
// Operands go from global memory straight into LDS with
// global_load_lds_dwordx4 (16 bytes per lane, 1 KB per wavefront
// instruction): no staging registers.  A K step is 64 wide, so every row of
// the A tile is one whole 128-byte line per step (measured on gfx950: copies
// of 64-byte row segments move half the bytes per clock that whole lines do).
// Two 64 KB stages: the copy of step s + 1 is issued in four slices
// interleaved with the MFMAs of step s (after the barrier that opens it).  The load side walks
// the tile sequence one step ahead of the compute side, across tile
// boundaries.  Everything else a tile needs from memory arrives by the same
// kind of copies: the gathered row indices of the next tile, the bias of
// the current one (it seeds the accumulators) and, for the weight gradient,
// the rows of the next stage (a plain load whose value is used would make
// the compiler wait for every copy in flight, which it does not see).  Lanes whose
// K element lies past the step's range copy from a page of zeros; in the
// forward product and the activation gradient, rows and columns past a
// tile's end read some other row or column of the operand instead (their
// products are never stored), so that a copy's source is one add away from
// a per-tile offset, and each 16-wide slice's copies sit between its MFMAs
// (a burst of copies ahead of them held the MFMAs back).
//
// LDS layouts, per stage:
//  * K-contiguous rows (X and dY rows, and W read as W^T): 128 bytes
//    (64 bf16) per row, the 16-byte chunk c of row r stored at chunk
//    c ^ ((r >> 1) & 7).  Eight lanes of a copy fill one row (the global side
//    reads the row's 128 contiguous bytes, permuted across lanes); a 32-row
//    MFMA operand read hits 16 distinct bank slots per 16 rows.
//  * N-contiguous rows (W in the forward product; X and dY rows in the
//    weight gradient, where K runs over positions): 64 K rows of 256 columns
//    (512 bytes), chunk c of K row k stored at chunk c ^ 4 (k & 3).  The
//    operand read uses ds_read_b64_tr_b16: in each 16-lane group, lanes
//    4r + q point at columns 4q..4q+3 of K row r and lane i receives column i
//    of those 4 rows, so two reads give a lane 8 consecutive K values of one
//    column, which is the MFMA operand layout.
#include <algorithm>
#include <type_traits>

#include "gemm_common.hpp"

namespace starq {

namespace {

using namespace gemm;

constexpr int kThreads = 512;                   // 8 wavefronts
constexpr int kWaves = kThreads / 64;
constexpr int BN = 256;                         // LDS column capacity of a B tile
constexpr int BK = 64;
constexpr int A_BYTES = BM * BK * 2;            // 256 rows x 64 bf16: 32 KB
constexpr int B_BYTES = BN * BK * 2;            // 256 columns x 64 bf16: 32 KB
constexpr int STAGE_BYTES = A_BYTES + B_BYTES;  // 64 KB
constexpr int SMEM = 2 * STAGE_BYTES;           // 128 KB
constexpr int DMA_A = A_BYTES / 1024 / kWaves;  // A copies per wave per stage (4)
constexpr int DMA_B = B_BYTES / 1024 / kWaves;  // B copies per wave per stage (4)
constexpr int kRowBufs = 4;                     // row-index / bias buffers

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

// wait until every vector-memory operation of this wave has completed
__device__ __forceinline__ void wait_vm_all() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));  // vmcnt(0)
  asm volatile("" ::: "memory");
}

__device__ __forceinline__ void block_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// whether the wave's rows, from tile row row0 on, hold any of a tile's
// `nrows` rows (uniform over the wave)
__device__ __forceinline__ bool wave_rows_live(int row0, int32_t nrows) {
  return __builtin_amdgcn_readfirstlane(row0 < nrows ? 1 : 0) != 0;
}

// Tile shapes: TM rows x TN columns, 8 wavefronts.  256 x 256: waves 2 x 4
// of 128 x 64; 256 x 192: waves 4 x 2 of 64 x 96 (groups 384 or 1536 wide
// take whole tiles); 192 x 256 (weight gradient only, rows over 384-wide
// input groups): waves 2 x 4 of 96 x 64.  The LDS tiles keep 256 rows and
// 256 columns of room either way.
template <int TM, int TN> struct Lay {
  static_assert((TM == 256 && (TN == 256 || TN == 192)) || (TM == 192 && TN == 256), "tile shape");
  static constexpr int WNW = TN == 256 ? 4 : 2;  // waves along N
  static constexpr int WMW = kWaves / WNW;        // waves along M
  static constexpr int TMW = TM / WMW;            // rows of a wave
  static constexpr int TNW = TN / WNW;            // columns of a wave
  static constexpr int MI = TMW / 32;             // 32-row MFMA blocks
  static constexpr int NI = TNW / 32;             // 32-column MFMA blocks
};

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return __builtin_amdgcn_readfirstlane(
      static_cast<uint32_t>(reinterpret_cast<uintptr_t>(p)));
}

// LDS reads are served 256 bytes (64 banks) at a time, 16 lanes of a 16-byte
// read or 32 lanes of an 8-byte read per pass.
// K-contiguous tile: byte offset of 16-byte chunk c of row r.  Rows r and
// r ^ 1 share a 256-byte bank line, so the chunk is rotated by (r >> 1) & 7:
// 16 consecutive rows at one chunk index cover all 16 bank slots.
__device__ __forceinline__ int kswz(int r) { return (r >> 1) & 7; }
__device__ __forceinline__ int krow_off(int r, int c) { return r * 128 + ((c ^ kswz(r)) << 4); }
// N-contiguous 256-column tile: byte offset of column chunk c of K row k.
// A transposing read covers 4 K rows x 4 chunks per 32 lanes; rotating the
// chunk by 4 (k & 3) puts them in 16 distinct bank slots.
__device__ __forceinline__ int kcol_off(int k, int c) { return k * 512 + ((c ^ (4 * (k & 3))) << 4); }

__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a, b}, bf16x2_t));
}

template <int MODE, int LAW, int ACT, int TM, int TN>
__global__ __launch_bounds__(kThreads, 1) void star_gemm_async_kernel(const GemmParams p) {
  static_assert(MODE == kModeBwdWeight || TM == BM, "tiles of fewer rows: weight gradient only");
  using L = Lay<TM, TN>;
  constexpr int MI = L::MI, NI = L::NI, TMW = L::TMW, TNW = L::TNW;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  // row tiles per class: [0] BM rows, [1] BM / 2 rows (weight gradient:
  // row tiles x splits, both)
  __shared__ int32_t units_s[2][kMaxQGroups];
  __shared__ int32_t offs_s[kMaxQGroups + 1];
  // tile prefix sums per class: pass 0, pass 1, pass 1 in half-height tiles
  __shared__ int32_t pfx_s[3][kMaxQGroups + 1];
  __shared__ __attribute__((aligned(16))) int32_t rows_s[kRowBufs][BM];
  __shared__ __attribute__((aligned(16))) float bias_s[kRowBufs][BN];
  // weight gradient: rows (perm entries) of the positions a stage contracts
  // over, two stages' worth
  __shared__ __attribute__((aligned(16))) int32_t prow_s[2][BK];

  const uint16_t* __restrict__ Ag = static_cast<const uint16_t*>(p.A);
  const uint16_t* __restrict__ Bg = static_cast<const uint16_t*>(p.B);
  const void* zero = g_zero_page;
  const int q = p.q;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave / L::WNW, wn = wave % L::WNW;
  const int lr = lane & 31, lh = lane >> 5;

  for (int i = threadIdx.x; i <= q; i += kThreads) offs_s[i] = p.offsets[i];
  __syncthreads();
  for (int i = threadIdx.x; i < q; i += kThreads) {
    if constexpr (MODE == kModeBwdWeight) {
      units_s[0][i] = units_s[1][i] = (p.MTp[i + 1] - p.MTp[i]) * p.nsplit;  // row tiles of K group i x splits
    } else {
      // row tiles of type class i
      units_s[0][i] = (offs_s[i + 1] - offs_s[i] + BM - 1) / BM;
      units_s[1][i] = (offs_s[i + 1] - offs_s[i] + BM / 2 - 1) / (BM / 2);
    }
  }
  __syncthreads();
  if (threadIdx.x < 3) {
    const int ps = threadIdx.x == 0 ? 0 : 1;
    const int sel = sel_for(MODE, LAW, ps);
    int32_t run = 0;
    for (int i = 0; i < q; ++i) {
      pfx_s[threadIdx.x][i] = run;
      run += units_s[threadIdx.x == 2 ? 1 : 0][i] * ncols_sel(p, sel, i);
    }
    pfx_s[threadIdx.x][q] = run;
  }
  __syncthreads();
  // Half-height tiles for pass 1 (star law) when whole tiles would deal out
  // unevenly: pass 0 fills at most one round of the grid, the two passes do
  // not fit in one, and so many pass-1 tiles remain that some workgroups get
  // a pass-0 and a pass-1 tile while the mean load is at least half a pass-1
  // tile below that (counted with equal groups, where a pass-0 tile has twice
  // the K steps of a pass-1 tile).  Half-height pass-1 tiles are dealt to the
  // workgroups without a pass-0 tile first; in such a tile the waves of the
  // empty half skip their MFMAs and epilogue.
  const int32_t n0 = pfx_s[0][q], n1 = pfx_s[1][q], ng = static_cast<int32_t>(gridDim.x);
  const int32_t whole_max = n1 > 2 * (ng - n0) ? 3 : 2;  // in pass-1 tiles
  const bool half1 =
      MODE != kModeBwdWeight && LAW == 0 &&
      __builtin_amdgcn_readfirstlane(n1 > 0 && n0 <= ng && n0 + n1 > ng &&
                                     2 * (whole_max * ng - 2 * n0 - n1) >= ng) != 0;
  const int p1 = half1 ? 2 : 1;  // the prefix sums pass 1 uses

  // ---- tile iterators (the compute side and the load side walk one list) ----
  // XCD x (workgroups w with w % 8 == x) owns a contiguous chunk of each
  // pass's tiles; its workgroups deal out the two chunks as one list, pass 0
  // (the longer contractions) first.
  const int xcd = blockIdx.x & 7;
  const int slot_stride = gridDim.x >> 3;
  int32_t pbase[2], pcount[2];
#pragma unroll
  for (int ps = 0; ps < 2; ++ps) {
    const int32_t total = pfx_s[ps == 0 ? 0 : p1][q];
    const int32_t chunk = (total + 7) >> 3;
    pbase[ps] = xcd * chunk;
    pcount[ps] = max(0, min(total - xcd * chunk, chunk));
  }
  // The XCD's workgroups take its list in snake order: in round r the
  // workgroup in place s (of S) takes item r S + s for even r and
  // r S + S - 1 - s for odd r, so a workgroup that got one of the first
  // (longest) items gets one of the last (shortest) ones if any.
  struct Iter {
    int32_t r;  // this workgroup's round
  };
  const int xslot = blockIdx.x >> 3;
  // With half-height pass-1 tiles, every round after the first runs in
  // reverse place order, so the half tiles go first to the workgroups that
  // had no pass-0 tile (the high places of round 0).
  auto advance = [&](Iter& it, Tile& t) -> bool {
    const bool rev = half1 ? it.r > 0 : (it.r & 1) != 0;
    const int32_t v = it.r * slot_stride + (rev ? slot_stride - 1 - xslot : xslot);
    if (v >= pcount[0] + pcount[1]) return false;
    ++it.r;
    const int ps = v < pcount[0] ? 0 : 1;
    const int32_t logical = pbase[ps] + (ps == 0 ? v : v - pcount[0]);
    const int32_t* pf = pfx_s[ps == 0 ? 0 : p1];
    int cls = 0;
    while (logical >= pf[cls + 1]) ++cls;
    const bool hh = ps == 1 && half1;
    t = make_tile<MODE, LAW, TN, BK>(p, sel_for(MODE, LAW, ps), cls, logical - pf[cls],
                                     units_s[hh ? 1 : 0][cls], offs_s, hh ? BM / 2 : TM);
    return true;
  };

  // weight gradient: a split whose row range is empty contributes zeros
  auto zero_tile = [&](const Tile& t) {
    float* out = p.nsplit > 1 ? p.partial + static_cast<int64_t>(t.split) * p.K * p.N : p.dW;
    for (int idx = threadIdx.x; idx < TM * TN / 4; idx += kThreads) {
      const int32_t r = t.rstart + idx / (TN / 4);
      const int32_t c = t.cstart + (idx % (TN / 4)) * 4;
      if (r < t.rend && c < t.cend)
        *reinterpret_cast<float4*>(out + static_cast<int64_t>(r) * p.N + c) = make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };

  Iter cit{0};
  Tile ct;
  if (!advance(cit, ct)) return;
  if constexpr (MODE == kModeBwdWeight) {
    while (ct.nsteps == 0) {
      zero_tile(ct);
      if (!advance(cit, ct)) return;
    }
  }

  // ---- load side: tile lt (sequence number lseq, step ls), next tile ln ----
  Iter lit = cit;
  Tile lt = ct, ln;
  int32_t lseq = 0, ls = 0;
  bool lvalid = true;
  bool rows_from_lds = false;  // rl must be refilled from rows_s
  // weight gradient: stage counter of the load side, and whether the rows
  // of each perm slot were copied ahead for the stage that will use it
  int32_t lstg = 0;
  uint32_t pok = 0;  // bit i: perm slot i holds the rows of the stage that will read it
  int32_t rl[DMA_A];  // gathered row of A copy j: tile row 8 (wave + 8 j) + lane / 8
#pragma unroll
  for (int j = 0; j < DMA_A; ++j) {
    const int row = 8 * (wave + kWaves * j) + (lane >> 3);
    rl[j] = row < lt.nrows ? p.perm[lt.pos0 + row] : -1;
  }
  // Copies of the forward product and the activation gradient: per tile,
  // the lane's A source of copy j (its row's base plus its 16-byte chunk; a
  // row past the tile's end reads row 0, whose products land in accumulator
  // rows that are never stored) and its B source relative to the step's B
  // base (forward: columns past the matrix end are clamped to its last 8;
  // activation gradient: rows of W past the tile's columns read its first
  // one; neither product is stored).  A step then adds one uniform offset
  // and tests one uniform length, so a copy is an add and a select.
  constexpr bool kFast = MODE != kModeBwdWeight;
  const int fa_chunk = (lane & 7) ^ ((4 * (wave & 1) + (lane >> 4)) & 7);  // K-contiguous chunk of every copy j
  const int fb_kr = 2 * wave + (lane >> 5);                                // forward B: K row of copy 0
  const int fb_chunk = (lane & 31) ^ (4 * (fb_kr & 3));                    // forward B: column chunk
  // (offsets in 16-byte units: K and N are multiples of 8, and the operands
  // are far below 64 GB)
  uint32_t aoff[DMA_A];
  uint32_t boff[MODE == kModeFwd ? 1 : DMA_B];
  // weight gradient: the lane's columns of X and of dY (its 16-byte chunk of
  // the tile's rows and columns of dW; chunks past the tile's end read
  // others, clamped into the matrix, whose products are not stored)
  int32_t wa_col = 0, wb_col = 0;
  auto tile_ptrs = [&]() {
    if constexpr (MODE == kModeBwdWeight) {
      wa_col = min(lt.rstart + 8 * (fb_chunk < TM / 8 ? fb_chunk : 0), p.K - 8);
      wb_col = min(lt.cstart + 8 * (fb_chunk < TN / 8 ? fb_chunk : 0), p.N - 8);
    }
    if constexpr (kFast) {
      const uint32_t lda8 = static_cast<uint32_t>((MODE == kModeFwd ? p.K : p.N) >> 3);
#pragma unroll
      for (int j = 0; j < DMA_A; ++j) aoff[j] = static_cast<uint32_t>(max(rl[j], 0)) * lda8 + fa_chunk;
      if constexpr (MODE == kModeFwd) {
        boff[0] = static_cast<uint32_t>(fb_kr) * static_cast<uint32_t>(p.N >> 3) +
                  static_cast<uint32_t>(min(fb_chunk < TN / 8 ? fb_chunk : 0, (p.N - 8 - lt.cstart) >> 3));
      } else {
#pragma unroll
        for (int j = 0; j < DMA_B; ++j) {
          const int row = 8 * (wave + kWaves * j) + (lane >> 3);
          const int32_t kk = lt.cstart + (lt.cstart + row < lt.cend ? row : 0);
          boff[j] = static_cast<uint32_t>(kk) * static_cast<uint32_t>(p.N >> 3) + fa_chunk;
        }
      }
    }
  };
  tile_ptrs();
  bool has_ln = advance(lit, ln);
  // the load side passes over tiles without K steps (weight-gradient splits
  // with empty row ranges); the compute side writes their zeros
  auto skip_empty = [&]() {
    if constexpr (MODE == kModeBwdWeight) {
      while (lvalid && lt.nsteps == 0) {
        if (has_ln) {
          lt = ln;
          has_ln = advance(lit, ln);
        } else {
          lvalid = false;
        }
      }
    }
  };

  // A stage is copied in three parts so that the copies can be spread over
  // the MFMAs of the step being computed: stage_begin picks the stage's K
  // range and issues the small copies (row indices of the next tile and
  // bias at a tile's first stage; the weight gradient's perm entries of the
  // next stage), copy_a(j) / copy_b(j) issue A copy j and B copy j of this
  // wave, stage_end moves the load side on.
  int32_t sk0 = 0, skend = 0, klen = 0;
  // LDS addresses of the load slot's A and B tiles (uniform: kept in scalar
  // registers, the copies' M0)
  const uint32_t lds0 = lds_addr(smem);
  uint32_t la = lds0, lb = lds0 + A_BYTES;
  const char* astep = reinterpret_cast<const char*>(Ag);  // forward: X at column sk0
  const char* bstep = reinterpret_cast<const char*>(Bg);  // forward: W at row sk0, column cstart of the load tile
  auto stage_begin = [&](int slot) {
    la = lds0 + slot * STAGE_BYTES;
    lb = la + A_BYTES;
    // past the last stage the copies repeat the previous step's sources
    // into the free slot
    if (!lvalid) return;
    if (rows_from_lds) {
      // ln's indices were copied with lt's first stage, which has landed
      // (every step waits for all copies in flight)
      if constexpr (kFast) {
#pragma unroll
        for (int j = 0; j < DMA_A; ++j) {
          const int row = 8 * (wave + kWaves * j) + (lane >> 3);
          rl[j] = row < lt.nrows ? rows_s[lseq & (kRowBufs - 1)][row] : -1;
        }
      }
      rows_from_lds = false;
      tile_ptrs();
    }
    step_range<MODE, LAW, BK>(p, lt, offs_s, ls, sk0, skend);
    klen = skend - sk0;
    if constexpr (kFast) {
      astep = reinterpret_cast<const char*>(Ag + sk0);
      bstep = MODE == kModeFwd ? reinterpret_cast<const char*>(Bg + static_cast<int64_t>(sk0) * p.N + lt.cstart)
                               : reinterpret_cast<const char*>(Bg + sk0);
      if (ls == 0) {
        if (wave < 4) {
          // row indices of the next tile
          const int r = 64 * wave + lane;
          const void* g = (has_ln && r < ln.nrows) ? static_cast<const void*>(p.perm + ln.pos0 + r) : zero;
          dma4(g, lds_addr(&rows_s[(lseq + 1) & (kRowBufs - 1)][64 * wave]));
        } else if (MODE == kModeFwd) {
          // bias of this tile's columns, 64 per wave
          const int32_t col = lt.cstart + 64 * (wave - 4) + lane;
          const void* g = (p.bias && col < lt.cend) ? static_cast<const void*>(p.bias + col) : zero;
          dma4(g, lds_addr(&bias_s[lseq & (kRowBufs - 1)][64 * (wave - 4)]));
        }
      }
    }
    if constexpr (MODE == kModeBwdWeight) {
      if (!((pok >> (lstg & 1)) & 1u)) {
        // the rows of this stage were not copied ahead (first stage, or the
        // tile after an empty one): fetch them now (nothing else is in
        // flight at a step's start)
        if (wave == 0) {
          const int32_t pos = sk0 + lane;
          dma4(pos < skend ? static_cast<const void*>(p.perm + pos) : zero, lds_addr(&prow_s[lstg & 1][0]));
        }
        wait_vm_all();
        block_barrier();
      }
      // this wave's rows for the stage's copies, read once (rl[j]: the row at
      // position sk0 + 2 (wave + 8 j) + lane / 32, or -1 past the range)
#pragma unroll
      for (int j = 0; j < DMA_A; ++j) {
        const int kr = 2 * (wave + kWaves * j) + (lane >> 5);
        rl[j] = sk0 + kr < skend ? prow_s[lstg & 1][kr] : -1;
      }
      // rows of the next stage, into the other perm slot (free: its last
      // reader was the previous step's start)
      int32_t nlo = 0, nhi = 0;
      bool next = false;
      if (ls + 1 < lt.nsteps) {
        step_range<MODE, LAW, BK>(p, lt, offs_s, ls + 1, nlo, nhi);
        next = true;
      } else if (has_ln && ln.nsteps > 0) {
        step_range<MODE, LAW, BK>(p, ln, offs_s, 0, nlo, nhi);
        next = true;
      }
      const uint32_t bit = 1u << ((lstg + 1) & 1);
      pok = next ? (pok | bit) : (pok & ~bit);
      if (next && wave == 0) {
        const int32_t npos = nlo + lane;
        dma4(npos < nhi ? static_cast<const void*>(p.perm + npos) : zero, lds_addr(&prow_s[(lstg + 1) & 1][0]));
      }
    }
  };
  // A copy j and B copy j of this wave.  Forward and activation gradient:
  // a uniform step offset and length, a select for the K tail.  Weight
  // gradient: A = X rows over the tile's K columns, B = dY rows over its N
  // columns, 2 positions of the type-sorted order per copy (rows read at the
  // step's start from the perm entries copied ahead), the zero page past
  // the step's range.
  auto copy_a = [&](int j) {
    const void* g;
    if constexpr (MODE == kModeBwdWeight) {
      g = rl[j] >= 0 ? static_cast<const void*>(Ag + static_cast<int64_t>(rl[j]) * p.K + wa_col) : zero;
    } else {
      const bool ok = 8 * fa_chunk < klen;
      g = ok ? static_cast<const void*>(astep + static_cast<uint64_t>(aoff[j]) * 16) : zero;
    }
    dma16(g, la + (wave + kWaves * j) * 1024);
  };
  auto copy_b = [&](int j) {
    const void* g;
    if constexpr (MODE == kModeBwdWeight) {
      g = rl[j] >= 0 ? static_cast<const void*>(Bg + static_cast<int64_t>(rl[j]) * p.N + wb_col) : zero;
    } else if constexpr (MODE == kModeFwd) {
      const bool ok = fb_kr + 2 * kWaves * j < klen;
      g = ok ? static_cast<const void*>(bstep + static_cast<int64_t>(2 * kWaves * j) * p.N * 2 +
                                        static_cast<uint64_t>(boff[0]) * 16)
             : zero;
    } else {
      // (rows of W past the tile width are not copied)
      if (j >= TN / 64) return;
      const bool ok = 8 * fa_chunk < klen;
      g = ok ? static_cast<const void*>(bstep + static_cast<uint64_t>(boff[j]) * 16) : zero;
    }
    dma16(g, lb + (wave + kWaves * j) * 1024);
  };
  auto stage_copy = [&](int j) {
    copy_a(j);
    copy_b(j);
  };
  auto stage_end = [&]() {
    if (!lvalid) return;
    ++lstg;
    if (++ls == lt.nsteps) {
      if (has_ln) {
        rows_from_lds = true;
        lt = ln;
        ++lseq;
        ls = 0;
        has_ln = advance(lit, ln);
        skip_empty();
      } else {
        lvalid = false;
      }
    }
  };
  static_assert(DMA_A == 4 && DMA_B == 4, "one A and one B copy per K slice of a step (fewer B copies at TN 192)");

  // fragments of one 16-wide K slice
  // 8 consecutive K values of one column from an N-contiguous tile, by two
  // transposing reads (K rows k and k + 4 of each 4 x 16 block)
  auto tr_frag = [&](const char* T, int k, int col) -> uint4 {
    const char* a0 = T + kcol_off(k, col >> 3) + ((col >> 2) & 1) * 8;
    const v4i16_t w0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((STARQ_LDS v4i16_t*)(a0));
    const v4i16_t w1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((STARQ_LDS v4i16_t*)(a0 + 4 * 512));
    uint4 f;
    f.x = static_cast<uint16_t>(w0[0]) | (static_cast<uint32_t>(static_cast<uint16_t>(w0[1])) << 16);
    f.y = static_cast<uint16_t>(w0[2]) | (static_cast<uint32_t>(static_cast<uint16_t>(w0[3])) << 16);
    f.z = static_cast<uint16_t>(w1[0]) | (static_cast<uint32_t>(static_cast<uint16_t>(w1[1])) << 16);
    f.w = static_cast<uint16_t>(w1[2]) | (static_cast<uint32_t>(static_cast<uint16_t>(w1[3])) << 16);
    return f;
  };
  auto read_frags = [&](const char* As, const char* Bs, int rs, uint4 (&fa)[MI], uint4 (&fb)[NI]) {
    if constexpr (MODE == kModeBwdWeight) {
      const int gq = lane >> 4, pp = lane & 15;
      const int k = 16 * rs + 8 * (gq >> 1) + (pp >> 2);
      const int cq = 16 * (gq & 1) + 4 * (pp & 3);
#pragma unroll
      for (int mi = 0; mi < MI; ++mi) fa[mi] = tr_frag(As, k, wm * TMW + mi * 32 + cq);
#pragma unroll
      for (int ni = 0; ni < NI; ++ni) fb[ni] = tr_frag(Bs, k, wn * TNW + ni * 32 + cq);
      return;
    }
    const int kp = 2 * rs + lh;
#pragma unroll
    for (int mi = 0; mi < MI; ++mi) {
      const int row = wm * TMW + mi * 32 + lr;
      fa[mi] = *reinterpret_cast<const uint4*>(As + krow_off(row, kp));
    }
    if constexpr (MODE == kModeFwd) {
      const int gq = lane >> 4, pp = lane & 15;
      const int k = 16 * rs + 8 * (gq >> 1) + (pp >> 2);
#pragma unroll
      for (int ni = 0; ni < NI; ++ni) {
        const int col = wn * TNW + ni * 32 + 16 * (gq & 1) + 4 * (pp & 3);
        const char* a0 = Bs + kcol_off(k, col >> 3) + ((col >> 2) & 1) * 8;
        const v4i16_t w0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((STARQ_LDS v4i16_t*)(a0));
        const v4i16_t w1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((STARQ_LDS v4i16_t*)(a0 + 4 * 512));
        fb[ni].x = static_cast<uint16_t>(w0[0]) | (static_cast<uint32_t>(static_cast<uint16_t>(w0[1])) << 16);
        fb[ni].y = static_cast<uint16_t>(w0[2]) | (static_cast<uint32_t>(static_cast<uint16_t>(w0[3])) << 16);
        fb[ni].z = static_cast<uint16_t>(w1[0]) | (static_cast<uint32_t>(static_cast<uint16_t>(w1[1])) << 16);
        fb[ni].w = static_cast<uint16_t>(w1[2]) | (static_cast<uint32_t>(static_cast<uint16_t>(w1[3])) << 16);
      }
    } else {
#pragma unroll
      for (int ni = 0; ni < NI; ++ni) {
        const int row = wn * TNW + ni * 32 + lr;
        fb[ni] = *reinterpret_cast<const uint4*>(Bs + krow_off(row, kp));
      }
    }
  };

  f32x16_t acc[MI][NI];
#pragma unroll
  for (int mi = 0; mi < MI; ++mi)
#pragma unroll
    for (int ni = 0; ni < NI; ++ni)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[mi][ni][e] = 0.f;

  // prologue: the first tile's rows for its epilogue, then stage 0
  if (MODE != kModeBwdWeight && wave < 4) {
    const int r = 64 * wave + lane;
    dma4(r < ct.nrows ? static_cast<const void*>(p.perm + ct.pos0 + r) : zero,
         lds_addr(&rows_s[0][64 * wave]));
  }
  skip_empty();
  stage_begin(0);
#pragma unroll
  for (int j = 0; j < DMA_A; ++j) stage_copy(j);
  stage_end();

  // first columns of the lane's groups of 4 consecutive outputs
  auto lcol = [&](int ni, int a) { return wn * TNW + ni * 32 + 8 * a + 4 * lh; };

  int32_t cseq = 0, cs = 0;
  int slot = 0;
  while (true) {
    wait_vm_all();    // this wave's copies for stage `slot` have landed
    block_barrier();  // and everyone's; the other slot (computed last step) is free
    stage_begin(slot ^ 1);
    if (cs == 0) {
      // a tile starts: the accumulators start from the bias (forward; its
      // copy came with this step's operands) or from zero
#pragma unroll
      for (int ni = 0; ni < NI; ++ni)
#pragma unroll
        for (int a = 0; a < 4; ++a) {
          float4 bv = make_float4(0.f, 0.f, 0.f, 0.f);
          if constexpr (MODE == kModeFwd) bv = *reinterpret_cast<const float4*>(&bias_s[cseq & (kRowBufs - 1)][lcol(ni, a)]);
#pragma unroll
          for (int mi = 0; mi < MI; ++mi) {
            acc[mi][ni][4 * a + 0] = bv.x;
            acc[mi][ni][4 * a + 1] = bv.y;
            acc[mi][ni][4 * a + 2] = bv.z;
            acc[mi][ni][4 * a + 3] = bv.w;
          }
        }
    }
    {
      const char* As = smem + slot * STAGE_BYTES;
      const char* Bs = As + A_BYTES;
      // a wave whose rows are all past the tile's rows (half-height tiles)
      // skips the MFMAs
      const bool wact = MODE == kModeBwdWeight || wave_rows_live(wm * TMW, ct.nrows);
      uint4 fa[2][MI], fb[2][NI];
      read_frags(As, Bs, 0, fa[0], fb[0]);
      {
        // The next stage's A and B copies of each 16-wide slice go between
        // its MFMAs (after the second and the fourth): issued in a burst
        // ahead of them, they held the MFMAs back.  The step is one block
        // either way (a wave whose rows are all past a half-height tile's
        // end runs the copies only).
        auto slices = [&](auto on) {
#pragma unroll
          for (int rs = 0; rs < 4; ++rs) {
            if (rs + 1 < 4) read_frags(As, Bs, rs + 1, fa[(rs + 1) & 1], fb[(rs + 1) & 1]);
#pragma unroll
            for (int x = 0; x < MI * NI; ++x) {
              if constexpr (decltype(on)::value)
                mma(acc[x / NI][x % NI], fb[rs & 1][x % NI], fa[rs & 1][x / NI], uint16_t());
              if (x == 1 || x == 3) {
                __builtin_amdgcn_sched_barrier(0);
                if (x == 1) copy_a(rs); else copy_b(rs);
                __builtin_amdgcn_sched_barrier(0);
              }
            }
          }
        };
        if (wact) slices(std::true_type{});
        else slices(std::false_type{});
      }
    }
    stage_end();
    slot ^= 1;
    if (++cs < ct.nsteps) continue;

    // ---- epilogue of tile ct ----
    if constexpr (MODE == kModeBwdWeight) {
      // dW rows k (C rows) x 4 consecutive columns n per lane group
      float* out = p.nsplit > 1 ? p.partial + static_cast<int64_t>(ct.split) * p.K * p.N : p.dW;
#pragma unroll
      for (int mi = 0; mi < MI; ++mi) {
        const int32_t k = ct.rstart + wm * TMW + mi * 32 + lr;
        float* yr = out + static_cast<int64_t>(k) * p.N + ct.cstart + wn * TNW + 4 * lh;
#pragma unroll
        for (int ni = 0; ni < NI; ++ni)
#pragma unroll
          for (int a = 0; a < 4; ++a)
            if (k < ct.rend && ct.cstart + wn * TNW + ni * 32 + 8 * a + 4 * lh < ct.cend)
              *reinterpret_cast<float4*>(yr + ni * 32 + 8 * a) =
                  make_float4(acc[mi][ni][4 * a], acc[mi][ni][4 * a + 1], acc[mi][ni][4 * a + 2],
                              acc[mi][ni][4 * a + 3]);
      }
    } else if (wave_rows_live(wm * TMW, ct.nrows))
    // The arithmetic runs over all the lane's accumulators without
    // control flow (so independent values interleave); only the memory
    // accesses are predicated on the row and column being inside the tile.
    {
      const int buf = cseq & (kRowBufs - 1);
      const int64_t ldc = (MODE == kModeFwd) ? p.N : p.K;
      bool rv[MI], cv[NI][4];
      int64_t rbase[MI];
#pragma unroll
      for (int mi = 0; mi < MI; ++mi) {
        const int row = wm * TMW + mi * 32 + lr;
        rv[mi] = row < ct.nrows;
        rbase[mi] = static_cast<int64_t>(rv[mi] ? rows_s[buf][row] : 0) * ldc + ct.cstart;
      }
#pragma unroll
      for (int ni = 0; ni < NI; ++ni)
#pragma unroll
        for (int a = 0; a < 4; ++a) cv[ni][a] = ct.cstart + lcol(ni, a) < ct.cend;
      // the bf16 stores write 8-column groups at ni * 32 + 16 pr of the
      // lane's columns (column ends are multiples of 8)
      const int clim8 = ct.cend - ct.cstart - wn * TNW - 8 * lh;

      // the lane's MI x NI x 4 groups of 4 consecutive outputs: one row
      // pointer per 32-row block, constant offsets for the rest
      auto store_tile = [&](void* out) {
        if (p.ydtype == 0) {
#pragma unroll
          for (int mi = 0; mi < MI; ++mi) {
            float* yr = static_cast<float*>(out) + rbase[mi] + wn * TNW + 4 * lh;
#pragma unroll
            for (int ni = 0; ni < NI; ++ni)
#pragma unroll
              for (int a = 0; a < 4; ++a)
                if (rv[mi] && cv[ni][a])
                  *reinterpret_cast<float4*>(yr + ni * 32 + 8 * a) =
                      make_float4(acc[mi][ni][4 * a], acc[mi][ni][4 * a + 1], acc[mi][ni][4 * a + 2],
                                  acc[mi][ni][4 * a + 3]);
          }
        } else {
          // Lanes l and l + 32 hold the two halves of each 8-column group:
          // one swap between the lane halves hands lane l all of group 2 pr
          // and lane l + 32 all of group 2 pr + 1, so every lane writes 16
          // bytes and a store covers 32 contiguous bytes of each of 32 rows
          // (half the store instructions of 8-byte pieces; measured 9 % off
          // the forward kernel at 8192 x 768 x 3072).
#pragma unroll
          for (int mi = 0; mi < MI; ++mi) {
            uint16_t* yr = static_cast<uint16_t*>(out) + rbase[mi] + wn * TNW;
#pragma unroll
            for (int ni = 0; ni < NI; ++ni)
#pragma unroll
              for (int pr = 0; pr < 2; ++pr) {
                const int a0 = 2 * pr, a1 = 2 * pr + 1;
                const auto sx = __builtin_amdgcn_permlane32_swap(
                    pack_bf16(acc[mi][ni][4 * a0], acc[mi][ni][4 * a0 + 1]),
                    pack_bf16(acc[mi][ni][4 * a1], acc[mi][ni][4 * a1 + 1]), false, false);
                const auto sy = __builtin_amdgcn_permlane32_swap(
                    pack_bf16(acc[mi][ni][4 * a0 + 2], acc[mi][ni][4 * a0 + 3]),
                    pack_bf16(acc[mi][ni][4 * a1 + 2], acc[mi][ni][4 * a1 + 3]), false, false);
                if (rv[mi] && ni * 32 + 16 * pr < clim8)
                  *reinterpret_cast<uint4*>(yr + ni * 32 + 8 * (a0 + lh)) = make_uint4(sx[0], sy[0], sx[1], sy[1]);
              }
          }
        }
      };
      if constexpr (MODE == kModeFwd) {
        // (the bias is already in: the accumulators started from it)
        if (p.Z) store_tile(p.Z);
        if constexpr (ACT != kActNone) {
#pragma unroll
          for (int mi = 0; mi < MI; ++mi)
#pragma unroll
            for (int ni = 0; ni < NI; ++ni)
#pragma unroll
              for (int e = 0; e < 16; ++e) acc[mi][ni][e] = act_apply(ACT, acc[mi][ni][e]);
        }
      } else if constexpr (ACT != kActNone) {
        // activation gradient: dX *= act'(Z_prev) at the same positions,
        // 4 values at a time (the fence keeps the compiler from hoisting
        // every Z_prev load and derivative, which would not fit in registers)
#pragma unroll
        for (int mi = 0; mi < MI; ++mi) {
          const uint16_t* zr = static_cast<const uint16_t*>(p.Zprev) + rbase[mi] + wn * TNW + 4 * lh;
#pragma unroll
          for (int ni = 0; ni < NI; ++ni)
#pragma unroll
            for (int a = 0; a < 4; ++a) {
              uint2 zw = make_uint2(0, 0);
              if (rv[mi] && cv[ni][a]) zw = *reinterpret_cast<const uint2*>(zr + ni * 32 + 8 * a);
              acc[mi][ni][4 * a + 0] *= act_deriv(ACT, bf16_to_f32(zw.x & 0xffffu));
              acc[mi][ni][4 * a + 1] *= act_deriv(ACT, bf16_to_f32(zw.x >> 16));
              acc[mi][ni][4 * a + 2] *= act_deriv(ACT, bf16_to_f32(zw.y & 0xffffu));
              acc[mi][ni][4 * a + 3] *= act_deriv(ACT, bf16_to_f32(zw.y >> 16));
              asm volatile("" ::: "memory");
            }
        }
      }
      store_tile(p.Y);
    }
    if (!advance(cit, ct)) break;
    if constexpr (MODE == kModeBwdWeight) {
      bool more = true;
      while (ct.nsteps == 0) {
        zero_tile(ct);
        if (!advance(cit, ct)) {
          more = false;
          break;
        }
      }
      if (!more) break;
    }
    ++cseq;
    cs = 0;
  }
  // every copy into LDS lands before the workgroup ends
  wait_vm_all();
}

template <int MODE, int LAW, int ACT, int TM, int TN>
hipError_t launch_one(const GemmParams& p, int64_t upper, int cus, hipStream_t stream) {
  auto kern = star_gemm_async_kernel<MODE, LAW, ACT, TM, TN>;
  static std::atomic<unsigned long long> lds_set{0};
  const hipError_t attr = ensure_lds_limit(reinterpret_cast<const void*>(kern), lds_set, SMEM);
  if (attr != hipSuccess) return attr;
  // persistent grid: one workgroup per CU, a multiple of 8 so that every
  // XCD gets the same number
  int64_t grid = std::min<int64_t>(std::max<int64_t>(upper, 1), static_cast<int64_t>(cus));
  grid = (grid + 7) / 8 * 8;
  hipLaunchKernelGGL(kern, dim3(static_cast<unsigned>(grid)), dim3(kThreads), SMEM, stream, p);
  return hipGetLastError();
}

// the 192-wide and 192-high tiles are built for the star and dense laws
// only, the 192-high ones for the weight gradient
template <int MODE, int LAW, int ACT>
hipError_t launch_tn(const GemmParams& p, int64_t upper, int cus, hipStream_t stream) {
  if constexpr (LAW <= 1) {
    if (p.tile_m == 256 && p.tile_n == 192) return launch_one<MODE, LAW, ACT, 256, 192>(p, upper, cus, stream);
    if constexpr (MODE == kModeBwdWeight) {
      if (p.tile_m == 192 && p.tile_n == 256) return launch_one<MODE, LAW, ACT, 192, 256>(p, upper, cus, stream);
    }
  }
  if (p.tile_m != 256 || p.tile_n != 256) return hipErrorInvalidValue;
  return launch_one<MODE, LAW, ACT, 256, 256>(p, upper, cus, stream);
}

template <int MODE, int LAW>
hipError_t launch_act(const GemmParams& p, int64_t upper, int cus, hipStream_t stream) {
  if constexpr (MODE == kModeBwdWeight) {
    return launch_tn<MODE, LAW, kActNone>(p, upper, cus, stream);
  } else {
    switch (p.act) {
      case kActGelu: return launch_tn<MODE, LAW, kActGelu>(p, upper, cus, stream);
      case kActGeluTanh: return launch_tn<MODE, LAW, kActGeluTanh>(p, upper, cus, stream);
      default: return launch_tn<MODE, LAW, kActNone>(p, upper, cus, stream);
    }
  }
}

template <int MODE>
hipError_t launch_async(const GemmParams& p, int64_t upper, int cus, hipStream_t stream) {
  if (p.law == 3) return launch_act<MODE, 3>(p, upper, cus, stream);
  if (p.law == 2) return launch_act<MODE, 2>(p, upper, cus, stream);
  return p.law == 1 ? launch_act<MODE, 1>(p, upper, cus, stream)
                    : launch_act<MODE, 0>(p, upper, cus, stream);
}

}  // namespace

hipError_t launch_gemm_async(int mode, const GemmParams& p, int64_t upper_tiles, int cus,
                             hipStream_t stream) {
  if (mode == kModeFwd) return launch_async<kModeFwd>(p, upper_tiles, cus, stream);
  if (mode == kModeBwdWeight) return launch_async<kModeBwdWeight>(p, upper_tiles, cus, stream);
  return launch_async<kModeBwdData>(p, upper_tiles, cus, stream);
}

}  // namespace starq
