// Grouped, row-typed GEMM on gfx950 MFMA for fp32 operands: the forward
// projection, its activation gradient and its weight gradient (Alg. 1 and
// the VJPs of the appendix) in one persistent kernel template.  bf16
// operands run in the pipelined kernel of gemm_async.hip.
//
// Work decomposition.  C is cut into tiles of 256 rows x BN columns
// (BN = 64 * WN, WN = 2).  A workgroup of 4 wavefronts (one per
// SIMD) computes a tile; the wavefronts form a 2 x 2 grid and each owns
// 128 x (32 * WN) of C as 4 x WN blocks of v_mfma_f32_32x32x16_bf16 (or of
// v_mfma_f32_32x32x2f32 for fp32 operands), accumulated in AGPRs.
//
//  * FWD: a tile is (row type i, row tile of I_i, output group j, column
//    tile).  Its K range is the concatenation of the input groups in
//    B(i,j): {j, i} for the star law (one group when j = i), all of K for
//    the dense law.  Rows are gathered through the type plan's permutation,
//    so each tile multiplies only rows that share one support: the skipped
//    blocks are never read and never multiplied.
//  * BWD_DATA: a tile is (row type i, row tile, input group g, column tile of
//    g).  Its contraction runs over the output groups j with g in B(i,j): all
//    of N when g = i (eq. vjp-xi), only group g otherwise (eq. vjp-xj).  W is
//    read in place as W^T (its rows are K-contiguous for this product).
//  * BWD_WEIGHT: a tile is (input group g, output group j, row tile of g,
//    column tile of j, split).  Its contraction runs over the rows whose
//    support reaches block (g, j): all rows when g = j (eqs. vjp-wii,
//    vjp-wjj), the type-g rows otherwise (eq. vjp-wij).  Long contractions
//    are split into a fixed number of row ranges whose fp32 partials a
//    second kernel sums in a fixed order.  The bias gradient is summed from
//    the dY tiles that the diagonal tiles already stage.
//
// Scheduling.  The kernel is persistent: one workgroup per CU walks its
// share of the tile list.  Tiles with the longer contraction come first
// (pass 0), the shorter ones after (pass 1).  Within a pass the list is cut
// into 8 contiguous chunks, one per XCD (workgroups are dispatched
// round-robin over the 8 XCDs), and consecutive tiles of a chunk share
// their weight panel, so the tiles running together on one XCD hit the same
// L2.  A workgroup runs its tiles as one flat sequence of K steps: while the
// last step of a tile computes, the first step of the next tile (whose row
// indices were fetched a whole tile earlier) is already being loaded.
//
// LDS layout.  Each K step stages 8 "kpacks" (16 bytes of K: 8 bf16 or 4
// fp32) per tile row, double-buffered.  A tile is stored kpack-major:
// unit (kp, row) holds the 16 bytes of K of that row, at
// (kp * rows + swz(row, kp)) * 16, where swz XORs the low three bits of the
// row with bits 3..5 of the row and the kpack index.  With it the three
// access patterns are free of bank conflicts: the MFMA operand read (32
// consecutive rows, one kpack), the direct store of K-contiguous rows
// (8 kpacks of one row from 8 lanes) and the transposed store.  Operands
// that are contiguous along the tile rows (W in the forward product, X and
// dY in the weight gradient) are transposed in registers on the way: each
// thread loads 4 source rows x 16 bytes and writes one 4-element piece per
// tile row.  Fragments for the next 16-wide K slice are read from LDS while
// the MFMAs of the current slice run.
//
// Epilogue.  The MFMA is issued with the operands swapped (it computes
// C^T blocks), so each lane ends with 4 consecutive columns of one row of
// C and writes them as one 8- or 16-byte store.  The activation and its
// derivative are the shared ones of common.hpp.
#include "gemm_common.hpp"

namespace starq {

namespace {

using namespace gemm;

// ---- operand staging -----------------------------------------------------

// K-contiguous source rows.  Unit u = tid + THREADS * i covers kpack u % 8
// of tile row u / 8 (8 lanes read one 128-byte row segment).
template <typename T, int ROWS>
struct DirectLoader {
  static constexpr int VEC = Tr<T>::VEC;
  static constexpr int UPT = ROWS * 8 / THREADS;
  static_assert(UPT * THREADS == ROWS * 8, "whole units per thread");
  uint4 reg[UPT];

  __device__ __forceinline__ static int row_of(int i) { return (threadIdx.x + THREADS * i) >> 3; }
  __device__ __forceinline__ static int kp_of() { return threadIdx.x & 7; }

  __device__ __forceinline__ void load(const T* __restrict__ src, int64_t ld, const int32_t* rowid,
                                       int32_t k0, int32_t kend) {
    const int32_t kk = k0 + kp_of() * VEC;
#pragma unroll
    for (int i = 0; i < UPT; ++i)
      reg[i] = load16(src, static_cast<int64_t>(rowid[i]) * ld + kk, rowid[i] >= 0 && kk < kend);
  }
  __device__ __forceinline__ void store(char* lds) const {
#pragma unroll
    for (int i = 0; i < UPT; ++i)
      *reinterpret_cast<uint4*>(lds + unit_off<ROWS>(kp_of(), row_of(i))) = reg[i];
  }
};

// Source contiguous along the tile rows (a source row is one K index).
// Block b = tid + THREADS * i covers source rows 4 q .. 4 q + 3 (q = b / CB)
// and tile rows VEC c .. VEC c + VEC - 1 (c = b % CB).
template <typename T, int ROWS>
struct TransLoader {
  static constexpr int VEC = Tr<T>::VEC;
  static constexpr int CB = ROWS / VEC;
  static constexpr int NQ = Tr<T>::BK / 4;
  static constexpr int BPT = CB * NQ / THREADS;
  static_assert(BPT * THREADS == CB * NQ, "whole blocks per thread");
  static_assert(THREADS % CB == 0, "a thread keeps its column chunk across blocks");
  uint4 reg[BPT][4];

  __device__ __forceinline__ static int cb_of() { return threadIdx.x % CB; }
  __device__ __forceinline__ static int q_of(int i) { return (threadIdx.x + THREADS * i) / CB; }

  template <typename RowFn>
  __device__ __forceinline__ void load(const T* __restrict__ src, int64_t ld, int32_t k0, int32_t c0,
                                       int32_t cend, RowFn srow) {
    const int32_t col = c0 + cb_of() * VEC;
#pragma unroll
    for (int i = 0; i < BPT; ++i) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int32_t row = srow(k0 + 4 * q_of(i) + e);
        reg[i][e] = load16(src, static_cast<int64_t>(row) * ld + col, row >= 0 && col < cend);
      }
    }
  }

  // optionally adds the staged values into per-column sums colsum[v]
  template <bool kSum>
  __device__ __forceinline__ void store(char* lds, float* colsum) const {
#pragma unroll
    for (int i = 0; i < BPT; ++i) {
      const int kbase = 4 * q_of(i);
      const int kp = kbase / VEC;
      const int boff = (kbase % VEC) * static_cast<int>(sizeof(T));
#pragma unroll
      for (int v = 0; v < VEC; ++v) {
        const int row = cb_of() * VEC + v;
        char* dst = lds + unit_off<ROWS>(kp, row) + boff;
        if constexpr (sizeof(T) == 2) {
          const int w = v >> 1, sh = (v & 1) * 16;
          const uint32_t e0 = (word_of(reg[i][0], w) >> sh) & 0xffffu;
          const uint32_t e1 = (word_of(reg[i][1], w) >> sh) & 0xffffu;
          const uint32_t e2 = (word_of(reg[i][2], w) >> sh) & 0xffffu;
          const uint32_t e3 = (word_of(reg[i][3], w) >> sh) & 0xffffu;
          *reinterpret_cast<uint2*>(dst) = make_uint2(e0 | (e1 << 16), e2 | (e3 << 16));
          if constexpr (kSum)
            colsum[v] += (bf16_to_f32(e0) + bf16_to_f32(e1)) + (bf16_to_f32(e2) + bf16_to_f32(e3));
        } else {
          const uint4 piece = make_uint4(word_of(reg[i][0], v), word_of(reg[i][1], v),
                                         word_of(reg[i][2], v), word_of(reg[i][3], v));
          *reinterpret_cast<uint4*>(dst) = piece;
          if constexpr (kSum)
            colsum[v] += (__uint_as_float(piece.x) + __uint_as_float(piece.y)) +
                         (__uint_as_float(piece.z) + __uint_as_float(piece.w));
        }
      }
    }
  }
};

template <int MODE, typename T, int WN> struct OperandLoaders;
template <typename T, int WN> struct OperandLoaders<kModeFwd, T, WN> {
  using A = DirectLoader<T, BM>;
  using B = TransLoader<T, Geo<WN>::BN>;
};
template <typename T, int WN> struct OperandLoaders<kModeBwdData, T, WN> {
  using A = DirectLoader<T, BM>;
  using B = DirectLoader<T, Geo<WN>::BN>;
};
template <typename T, int WN> struct OperandLoaders<kModeBwdWeight, T, WN> {
  using A = TransLoader<T, BM>;
  using B = TransLoader<T, Geo<WN>::BN>;
};

// Eight K steps of 16 (bf16) or 8 (fp32) per LDS stage: 4 slices, each one
// kpack per lane half.  Fragments of slice rs + 1 are read while the MFMAs
// of slice rs issue.
template <typename T, int WN>
__device__ __forceinline__ void compute_step(const char* As, const char* Bs, f32x16_t (&acc)[4][WN]) {
  constexpr int BN = Geo<WN>::BN;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int lr = lane & 31, lh = lane >> 5;
  uint4 fa[2][4], fb[2][WN];
  auto read = [&](int rs, int set) {
    const int kp = 2 * rs + lh;
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
      fa[set][mi] = *reinterpret_cast<const uint4*>(As + unit_off<BM>(kp, wm * 128 + mi * 32 + lr));
#pragma unroll
    for (int ni = 0; ni < WN; ++ni)
      fb[set][ni] = *reinterpret_cast<const uint4*>(Bs + unit_off<BN>(kp, wn * (32 * WN) + ni * 32 + lr));
  };
  read(0, 0);
#pragma unroll
  for (int rs = 0; rs < 4; ++rs) {
    if (rs + 1 < 4) read(rs + 1, (rs + 1) & 1);
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
      for (int ni = 0; ni < WN; ++ni) mma(acc[mi][ni], fb[rs & 1][ni], fa[rs & 1][mi], T());
  }
  // Pin the pipeline order for the scheduler: the reads of slice 0 and 1,
  // then each slice's MFMAs followed by the reads of the slice after next.
  constexpr int kReads = 4 + WN;
  constexpr int kMfma = 4 * WN * (sizeof(T) == 2 ? 1 : 4);
  __builtin_amdgcn_sched_group_barrier(0x100, 2 * kReads, 0);
#pragma unroll
  for (int rs = 0; rs < 4; ++rs) {
    __builtin_amdgcn_sched_group_barrier(0x008, kMfma, 0);
    if (rs + 2 < 4) __builtin_amdgcn_sched_group_barrier(0x100, kReads, 0);
  }
}

// Gathered row indices a thread needs for one FWD/BWD_DATA tile: the rows
// of its direct A loads and the rows its epilogue writes.
template <int UPT>
struct Rows {
  int32_t a[UPT];
  int32_t e[4];
};

template <int UPT>
__device__ __forceinline__ void fetch_rows(const GemmParams& p, const Tile& t, Rows<UPT>& r) {
  const int lane = threadIdx.x & 63;
  const int wm = (threadIdx.x >> 6) >> 1;
#pragma unroll
  for (int i = 0; i < UPT; ++i) {
    const int row = (threadIdx.x + THREADS * i) >> 3;
    r.a[i] = row < t.nrows ? p.perm[t.pos0 + row] : -1;
  }
#pragma unroll
  for (int mi = 0; mi < 4; ++mi) {
    const int row = wm * 128 + mi * 32 + (lane & 31);
    r.e[mi] = row < t.nrows ? p.perm[t.pos0 + row] : -1;
  }
}

template <typename T, int MODE, int LAW, int WN>
__global__ __launch_bounds__(THREADS, 1) void star_gemm_kernel(const GemmParams p) {
  using G = Geo<WN>;
  using LA = typename OperandLoaders<MODE, T, WN>::A;
  using LB = typename OperandLoaders<MODE, T, WN>::B;
  constexpr int BK = Tr<T>::BK;
  constexpr int BN = G::BN;
  constexpr int VEC = Tr<T>::VEC;
  constexpr int UPT = DirectLoader<T, BM>::UPT;  // row ids of the gathered A rows
  constexpr int BUPT = DirectLoader<T, BN>::UPT;   // BWD_DATA: rows of W per thread
  extern __shared__ __attribute__((aligned(16))) char smem[];
  __shared__ int32_t units_s[kMaxQGroups];
  __shared__ int32_t pfx_s[2][kMaxQGroups + 1];

  auto As = [&](int buf) { return smem + buf * G::STAGE; };
  auto Bs = [&](int buf) { return smem + buf * G::STAGE + G::A_BYTES; };
  const T* __restrict__ Ag = static_cast<const T*>(p.A);
  const T* __restrict__ Bg = static_cast<const T*>(p.B);
  const int q = p.q;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int lr = lane & 31, lh = lane >> 5;

  for (int i = threadIdx.x; i < q; i += THREADS) {
    if constexpr (MODE == kModeBwdWeight) {
      units_s[i] = (p.MTp[i + 1] - p.MTp[i]) * p.nsplit;
    } else {
      const int32_t mi = p.offsets[i + 1] - p.offsets[i];
      units_s[i] = (mi + BM - 1) / BM;
    }
  }
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

  // ---- this workgroup's tile sequence ----
  const int xcd = blockIdx.x & 7;
  const int slot_stride = gridDim.x >> 3;
  int it_pass = 0;
  int32_t it_slot = blockIdx.x >> 3;

  // zero tile of a weight-gradient split with an empty row range
  auto write_zero_tile = [&](const Tile& t) {
    float* out = p.nsplit > 1 ? p.partial + static_cast<int64_t>(t.split) * p.K * p.N : p.dW;
    for (int idx = threadIdx.x; idx < BM * BN / 4; idx += THREADS) {
      const int32_t r = t.rstart + idx / (BN / 4);
      const int32_t c = t.cstart + (idx % (BN / 4)) * 4;
      if (r < t.rend && c < t.cend)
        *reinterpret_cast<float4*>(out + static_cast<int64_t>(r) * p.N + c) = make_float4(0, 0, 0, 0);
    }
    if (t.do_dbias) {
      for (int c = threadIdx.x; c < BN; c += THREADS) {
        const int32_t gc = t.cstart + c;
        if (gc < t.cend) {
          if (p.nsplit > 1) p.dbias_part[static_cast<int64_t>(t.split) * p.N + gc] = 0.f;
          else p.dbias[gc] = 0.f;
        }
      }
    }
  };

  auto advance = [&](Tile& t) -> bool {
    while (it_pass < 2) {
      const int32_t total = pfx_s[it_pass][q];
      const int32_t chunk = (total + 7) >> 3;
      const int32_t logical = xcd * chunk + it_slot;
      if (it_slot >= chunk || logical >= total) {
        ++it_pass;
        it_slot = blockIdx.x >> 3;
        continue;
      }
      it_slot += slot_stride;
      int cls = 0;
      while (logical >= pfx_s[it_pass][cls + 1]) ++cls;
      const int sel = sel_for(MODE, LAW, it_pass);
      t = make_tile<MODE, LAW, BN, BK>(p, sel, cls, logical - pfx_s[it_pass][cls], units_s[cls],
                                       p.offsets);
      if (t.nsteps == 0) {  // only weight-gradient splits can be empty
        write_zero_tile(t);
        continue;
      }
      return true;
    }
    return false;
  };

  Tile cur, nxt;
  if (!advance(cur)) return;
  bool has_nxt = advance(nxt);
  Rows<UPT> rc, rn;
  if constexpr (MODE != kModeBwdWeight) {
    fetch_rows(p, cur, rc);
    if (has_nxt) fetch_rows(p, nxt, rn);
  }
  int32_t brow[BUPT];
  float colsum[VEC], colsum_n[VEC];
#pragma unroll
  for (int v = 0; v < VEC; ++v) colsum[v] = colsum_n[v] = 0.f;

  LA la;
  LB lb;
  // stage s of tile t into the loader registers
  auto load_stage = [&](const Tile& t, const Rows<UPT>& r, int32_t s) {
    int32_t k0, kend;
    step_range<MODE, LAW, BK>(p, t, p.offsets, s, k0, kend);
    if constexpr (MODE == kModeFwd) {
      la.load(Ag, p.K, r.a, k0, kend);
      lb.load(Bg, p.N, k0, t.cstart, t.cend, [&](int32_t k) { return k < kend ? k : -1; });
    } else if constexpr (MODE == kModeBwdData) {
#pragma unroll
      for (int i = 0; i < BUPT; ++i) {
        const int32_t kk = t.cstart + DirectLoader<T, BN>::row_of(i);
        brow[i] = kk < t.cend ? kk : -1;
      }
      la.load(Ag, p.N, r.a, k0, kend);
      lb.load(Bg, p.N, brow, k0, kend);
    } else {
      const int32_t* __restrict__ perm = p.perm;
      auto srow = [&](int32_t k) { return k < kend ? perm[k] : -1; };
      la.load(Ag, p.K, k0, t.rstart, t.rend, srow);
      lb.load(Bg, p.N, k0, t.cstart, t.cend, srow);
    }
  };
  auto store_stage = [&](int buf, bool dbias, float* cs) {
    if constexpr (MODE == kModeFwd) {
      la.store(As(buf));
      lb.template store<false>(Bs(buf), cs);
    } else if constexpr (MODE == kModeBwdData) {
      la.store(As(buf));
      lb.store(Bs(buf));
    } else {
      la.template store<false>(As(buf), cs);
      if (dbias) lb.template store<true>(Bs(buf), cs);
      else lb.template store<false>(Bs(buf), cs);
    }
  };

  load_stage(cur, rc, 0);
  store_stage(0, cur.do_dbias, colsum);  // colsum starts at zero
  __syncthreads();

  int buf = 0;
  while (true) {
    f32x16_t acc[4][WN];
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
      for (int ni = 0; ni < WN; ++ni)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[mi][ni][e] = 0.f;

    for (int32_t s = 0; s < cur.nsteps; ++s) {
      // the next stage: step s + 1 of this tile, or step 0 of the next one
      const bool more = s + 1 < cur.nsteps;
      const bool next_stage = more || has_nxt;
      const Tile lt = more ? cur : nxt;
      if (next_stage) {
        Rows<UPT> lrow;
#pragma unroll
        for (int i = 0; i < UPT; ++i) lrow.a[i] = more ? rc.a[i] : rn.a[i];
        load_stage(lt, lrow, more ? s + 1 : 0);
      }
      compute_step<T, WN>(As(buf), Bs(buf), acc);
      if (next_stage) {
        float cs[VEC];
#pragma unroll
        for (int v = 0; v < VEC; ++v) cs[v] = 0.f;
        store_stage(buf ^ 1, lt.do_dbias, cs);
        if constexpr (MODE == kModeBwdWeight) {
#pragma unroll
          for (int v = 0; v < VEC; ++v) {
            colsum[v] += more ? cs[v] : 0.f;
            colsum_n[v] += more ? 0.f : cs[v];
          }
        }
      }
      __syncthreads();
      buf ^= 1;
    }
    // `buf` now holds the next tile's first stage; `buf ^ 1` is free until
    // the next store into it

    // ---- epilogue of `cur` ----
    // lane holds C[row m][columns n .. n+3] with m = wm*128 + mi*32 + lr and
    // n = wn*32*WN + ni*32 + 8a + 4lh, values acc[mi][ni][4a .. 4a+3]
    if constexpr (MODE == kModeFwd || MODE == kModeBwdData) {
      const int64_t ldc = (MODE == kModeFwd) ? p.N : p.K;
#pragma unroll
      for (int mi = 0; mi < 4; ++mi) {
        const int32_t grow = rc.e[mi];
        if (grow < 0) continue;
#pragma unroll
        for (int ni = 0; ni < WN; ++ni)
#pragma unroll
          for (int a = 0; a < 4; ++a) {
            const int32_t gcol = cur.cstart + wn * (32 * WN) + ni * 32 + 8 * a + 4 * lh;
            if (gcol >= cur.cend) continue;
            const int64_t idx = static_cast<int64_t>(grow) * ldc + gcol;
            float v[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) v[j] = acc[mi][ni][4 * a + j];
            if constexpr (MODE == kModeFwd) {
              if (p.bias) {
                const float4 bv = *reinterpret_cast<const float4*>(p.bias + gcol);
                v[0] += bv.x; v[1] += bv.y; v[2] += bv.z; v[3] += bv.w;
              }
              if (p.Z) store4(p.Z, p.ydtype, idx, v);
              if (p.act != kActNone) {
#pragma unroll
                for (int j = 0; j < 4; ++j) v[j] = act_apply(p.act, v[j]);
              }
            } else {
              if (p.Zprev) {
                float z[4];
                load4(p.Zprev, p.elem == 0 ? 0 : 1, idx, z);
#pragma unroll
                for (int j = 0; j < 4; ++j) v[j] *= act_deriv(p.act, z[j]);
              }
            }
            store4(p.Y, p.ydtype, idx, v);
          }
      }
    } else {
      float* out = p.nsplit > 1 ? p.partial + static_cast<int64_t>(cur.split) * p.K * p.N : p.dW;
#pragma unroll
      for (int mi = 0; mi < 4; ++mi) {
        const int32_t grow = cur.rstart + wm * 128 + mi * 32 + lr;
        if (grow >= cur.rend) continue;
#pragma unroll
        for (int ni = 0; ni < WN; ++ni)
#pragma unroll
          for (int a = 0; a < 4; ++a) {
            const int32_t gcol = cur.cstart + wn * (32 * WN) + ni * 32 + 8 * a + 4 * lh;
            if (gcol >= cur.cend) continue;
            *reinterpret_cast<float4*>(out + static_cast<int64_t>(grow) * p.N + gcol) =
                make_float4(acc[mi][ni][4 * a], acc[mi][ni][4 * a + 1], acc[mi][ni][4 * a + 2],
                            acc[mi][ni][4 * a + 3]);
          }
      }
      if (cur.do_dbias) {
        // column sums of the staged dY: a thread keeps one column chunk;
        // reduce over the threads sharing it through LDS (free stage buffer)
        constexpr int kSlots = THREADS / LB::CB;
        float* red = reinterpret_cast<float*>(As(buf ^ 1));
        const int cb = LB::cb_of();
        const int slotr = threadIdx.x / LB::CB;
#pragma unroll
        for (int v = 0; v < VEC; ++v) red[slotr * BN + cb * VEC + v] = colsum[v];
        __syncthreads();
        for (int c = threadIdx.x; c < BN; c += THREADS) {
          float sum = 0.f;
          for (int sl = 0; sl < kSlots; ++sl) sum += red[sl * BN + c];
          const int32_t gcol = cur.cstart + c;
          if (gcol < cur.cend) {
            if (p.nsplit > 1) p.dbias_part[static_cast<int64_t>(cur.split) * p.N + gcol] = sum;
            else p.dbias[gcol] = sum;
          }
        }
        __syncthreads();
      }
    }

    if (!has_nxt) break;
    cur = nxt;
    rc = rn;
#pragma unroll
    for (int v = 0; v < VEC; ++v) {
      colsum[v] = colsum_n[v];
      colsum_n[v] = 0.f;
    }
    has_nxt = advance(nxt);
    if constexpr (MODE != kModeBwdWeight) {
      if (has_nxt) fetch_rows(p, nxt, rn);
    }
  }
}

// out = sum over s of part[s], in split order (so the result does not depend
// on timing).  The partials of up to 8 splits are loaded together before
// any is added: one dependent load after another left each thread waiting
// out nsplit memory round trips.
__global__ void split_reduce_kernel(const float* __restrict__ part, int nsplit, int64_t n,
                                    float* __restrict__ out) {
  const int64_t n4 = n >> 2;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n4;
       i += (int64_t)gridDim.x * blockDim.x) {
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int s0 = 0; s0 < nsplit; s0 += 8) {
      float4 v[8];
#pragma unroll
      for (int k = 0; k < 8; ++k)
        v[k] = s0 + k < nsplit ? reinterpret_cast<const float4*>(part + static_cast<int64_t>(s0 + k) * n)[i]
                               : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        if (s0 + k < nsplit) {
          acc.x += v[k].x; acc.y += v[k].y; acc.z += v[k].z; acc.w += v[k].w;
        }
      }
    }
    reinterpret_cast<float4*>(out)[i] = acc;
  }
  // tail (n not a multiple of 4)
  const int64_t t = (n4 << 2) + blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (blockIdx.x == 0 && t < n) {
    float a = part[t];
    for (int s = 1; s < nsplit; ++s) a += part[static_cast<int64_t>(s) * n + t];
    out[t] = a;
  }
}

__global__ void fill_zero_kernel(float* __restrict__ dst, int64_t n) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = 0.f;
}

template <typename T, int MODE, int WN, int LAW>
hipError_t launch_law(const GemmParams& p, int grid, hipStream_t stream) {
  using G = Geo<WN>;
  auto kern = star_gemm_kernel<T, MODE, LAW, WN>;
  // allow more than the default dynamic LDS (once per kernel and device)
  static std::atomic<unsigned long long> lds_set{0};
  const hipError_t attr = ensure_lds_limit(reinterpret_cast<const void*>(kern), lds_set, G::SMEM);
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL(kern, dim3(grid), dim3(THREADS), G::SMEM, stream, p);
  return hipGetLastError();
}

template <typename T, int MODE, int WN>
hipError_t launch_typed(const GemmParams& p, int grid, hipStream_t stream) {
  switch (p.law) {
    case 1: return launch_law<T, MODE, WN, 1>(p, grid, stream);
    case 2: return launch_law<T, MODE, WN, 2>(p, grid, stream);
    case 3: return launch_law<T, MODE, WN, 3>(p, grid, stream);
    default: return launch_law<T, MODE, WN, 0>(p, grid, stream);
  }
}

// fp32 operands only: bf16 operands run in the pipelined kernel.
template <int MODE, int WN>
hipError_t launch_mode(const GemmParams& p, int grid, hipStream_t stream) {
  if (p.elem != 0) return hipErrorInvalidValue;
  return launch_typed<float, MODE, WN>(p, grid, stream);
}

}  // namespace

hipError_t launch_gemm(int mode, const GemmParams& p, int nw, int grid, hipStream_t stream) {
  if (nw != 2) return hipErrorInvalidValue;
  if (mode == kModeFwd) return launch_mode<kModeFwd, 2>(p, grid, stream);
  if (mode == kModeBwdData) return launch_mode<kModeBwdData, 2>(p, grid, stream);
  return launch_mode<kModeBwdWeight, 2>(p, grid, stream);
}

hipError_t launch_fill_zero(float* dst, int64_t n, hipStream_t stream) {
  const int blocks = static_cast<int>(std::min<int64_t>(1024, (n + 255) / 256 + 1));
  hipLaunchKernelGGL(fill_zero_kernel, dim3(blocks), dim3(256), 0, stream, dst, n);
  return hipGetLastError();
}

hipError_t launch_sum_partials(const float* part, int n_parts, int64_t n, float* out,
                               hipStream_t stream) {
  const int blocks = static_cast<int>(std::min<int64_t>(2048, (n / 4 + 255) / 256 + 1));
  hipLaunchKernelGGL(split_reduce_kernel, dim3(blocks), dim3(256), 0, stream, part, n_parts, n, out);
  return hipGetLastError();
}

hipError_t launch_split_reduce(const GemmParams& p, hipStream_t stream) {
  const int64_t nKN = static_cast<int64_t>(p.K) * p.N;
  int blocks = static_cast<int>(std::min<int64_t>(2048, (nKN / 4 + 255) / 256 + 1));
  hipLaunchKernelGGL(split_reduce_kernel, dim3(blocks), dim3(256), 0, stream, p.partial,
                     p.nsplit, nKN, p.dW);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.dbias == nullptr) return e;
  return launch_sum_chunks(p.dbias_part, p.nsplit, p.N, p.dbias, stream);
}

}  // namespace starq
