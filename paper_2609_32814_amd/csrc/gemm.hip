// Grouped, row-typed GEMM on gfx950 MFMA: the forward projection, its
// activation gradient and its weight gradient (Alg. 1 and the VJPs of the
// appendix) in one persistent kernel template.
//
// Work decomposition.  C is tiled in 128 x 128 tiles, one per workgroup
// iteration (256 threads = 4 wavefronts in a 2 x 2 arrangement, 64 x 64 of
// C per wavefront as 2 x 2 blocks of v_mfma_f32_32x32x16_bf16, or of
// v_mfma_f32_32x32x2f32 for fp32 operands).
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
// Scheduling.  The kernel is persistent: a grid of about two workgroups per
// CU walks the tile list.  Tiles with the longer contraction run first
// (pass 0), the shorter ones after (pass 1).  Within a pass the list is cut
// into 8 contiguous chunks, one per XCD (workgroups are dispatched
// round-robin over the 8 XCDs), and consecutive tiles of a chunk share their
// weight panel, so concurrently running tiles of one XCD hit the same L2.
//
// Operand staging.  Each K step moves 128 bytes of K per row into LDS
// (64 bf16 or 32 fp32), double-buffered with one barrier per step.  Operands
// whose rows are K-contiguous are copied 16 bytes per lane; operands that are
// contiguous along the output dimension (W in the forward product, X and dY
// in the weight gradient) are transposed in registers on their way into LDS
// (each lane loads 4 bf16 rows x 8 columns, or 2 fp32 rows x 4 columns, and
// writes 8-byte K-contiguous pieces), so every MFMA operand is read from LDS
// as one 16-byte vector per lane.
#include "common.hpp"
#include "kernels.hpp"

namespace starq {

namespace {

constexpr int BM = kTileM;
constexpr int BN = kTileN;
constexpr int kThreads = kGemmThreads;
constexpr int kRowBytes = 144;  // 128 bytes of K + 16 bytes of padding
constexpr int kTileBytes = BM * kRowBytes;
static_assert(BM == BN, "A and B LDS tiles share one layout");
constexpr int kSmemBytes = 4 * kTileBytes;  // A and B, double-buffered

enum Sel : int { kSelNone = 0, kSelOnly = 1, kSelExcept = 2, kSelAll = 3 };

template <typename T> struct Traits;
template <> struct Traits<float> {
  static constexpr int VEC = 4;  // elements per 16-byte vector
  static constexpr int BK = 32;  // K per step (128 bytes)
  static constexpr int TK = 2;   // K rows per transposed 8-byte LDS write
};
template <> struct Traits<uint16_t> {
  static constexpr int VEC = 8;
  static constexpr int BK = 64;
  static constexpr int TK = 4;
};

__device__ __forceinline__ uint32_t word_of(const uint4& r, int w) {
  return w == 0 ? r.x : (w == 1 ? r.y : (w == 2 ? r.z : r.w));
}

__device__ __forceinline__ int sel_for(int mode, int law, int pass) {
  if (law == 1) return pass == 0 ? kSelAll : kSelNone;
  if (mode == kModeFwd) return pass == 0 ? kSelExcept : kSelOnly;
  return pass == 0 ? kSelOnly : kSelExcept;  // BWD_DATA and BWD_WEIGHT
}

__device__ __forceinline__ int ncols_sel(const GemmParams& p, int sel, int i) {
  const int nti = p.NTp[i + 1] - p.NTp[i];
  const int nt = p.NTp[p.q];
  switch (sel) {
    case kSelOnly: return nti;
    case kSelExcept: return nt - nti;
    case kSelAll: return nt;
    default: return 0;
  }
}

__device__ __forceinline__ int col_tile_global(const GemmParams& p, int sel, int i, int c) {
  if (sel == kSelOnly) return p.NTp[i] + c;
  if (sel == kSelExcept) return c < p.NTp[i] ? c : c + (p.NTp[i + 1] - p.NTp[i]);
  return c;
}

__device__ __forceinline__ void mma(f32x16_t& acc, const uint4& a, const uint4& b, uint16_t) {
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                __builtin_bit_cast(bf16x8_t, b), acc, 0, 0, 0);
}

__device__ __forceinline__ void mma(f32x16_t& acc, const uint4& a, const uint4& b, float) {
  // lane half h supplies K elements 4h..4h+3 of this 8-wide slice, one per
  // instruction; A and B use the same assignment, so the products pair up.
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
}

// ---- operand staging -------------------------------------------------------

// K-contiguous rows: LDS row r <- src[rowid[r]][k0 .. k0+BK), zero outside
// [.., kend) or for rowid < 0.  Thread t covers rows t/8 + 32u, 16-byte
// chunk t%8.
template <typename T>
__device__ __forceinline__ void load_k(uint4 (&reg)[4], const T* __restrict__ src, int64_t ld,
                                       const int32_t (&rowid)[4], int32_t k0, int32_t kend) {
  constexpr int VEC = Traits<T>::VEC;
  const int32_t kk = k0 + (threadIdx.x & 7) * VEC;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    if (rowid[u] >= 0 && kk < kend)
      reg[u] = *reinterpret_cast<const uint4*>(src + static_cast<int64_t>(rowid[u]) * ld + kk);
    else
      reg[u] = make_uint4(0, 0, 0, 0);
  }
}

__device__ __forceinline__ void store_k(char* lds, const uint4 (&reg)[4]) {
#pragma unroll
  for (int u = 0; u < 4; ++u)
    *reinterpret_cast<uint4*>(lds + ((threadIdx.x >> 3) + 32 * u) * kRowBytes +
                              (threadIdx.x & 7) * 16) = reg[u];
}

// Output-contiguous source: LDS row c (a column of the source) <- source
// rows k0 .. k0+BK at column c0 + c.  Source row of K index k is
// srow(k) (or < 0 to zero it).
template <typename T> struct TGeom {
  static constexpr int VEC = Traits<T>::VEC;
  static constexpr int TK = Traits<T>::TK;
  static constexpr int CB = BN / VEC;              // column chunks
  static constexpr int KB = Traits<T>::BK / TK;    // K pieces
  static constexpr int BPT = CB * KB / kThreads;   // blocks per thread
  static_assert(BPT * TK == 4, "four 16-byte staging registers per operand");
};

template <typename T, typename RowFn>
__device__ __forceinline__ void load_t(uint4 (&reg)[4], const T* __restrict__ src, int64_t ld,
                                       int32_t k0, int32_t c0, int32_t cend, RowFn srow) {
  using G = TGeom<T>;
#pragma unroll
  for (int blk = 0; blk < G::BPT; ++blk) {
    const int b = threadIdx.x + kThreads * blk;
    const int cb = b % G::CB;
    const int kb = b / G::CB;
    const int32_t col = c0 + cb * G::VEC;
#pragma unroll
    for (int e = 0; e < G::TK; ++e) {
      const int32_t row = srow(k0 + kb * G::TK + e);
      if (row >= 0 && col < cend)
        reg[blk * G::TK + e] =
            *reinterpret_cast<const uint4*>(src + static_cast<int64_t>(row) * ld + col);
      else
        reg[blk * G::TK + e] = make_uint4(0, 0, 0, 0);
    }
  }
}

// Transposed write of the staged blocks; optionally adds every staged value
// into per-column sums (colsum[v] for column chunk cb, element v).
template <typename T, bool kSum>
__device__ __forceinline__ void store_t(char* lds, const uint4 (&reg)[4], float* colsum) {
  using G = TGeom<T>;
#pragma unroll
  for (int blk = 0; blk < G::BPT; ++blk) {
    const int b = threadIdx.x + kThreads * blk;
    const int cb = b % G::CB;
    const int kb = b / G::CB;
#pragma unroll
    for (int v = 0; v < G::VEC; ++v) {
      uint2 piece;
      if constexpr (sizeof(T) == 2) {
        const int w = v >> 1;
        const int sh = (v & 1) * 16;
        const uint32_t e0 = (word_of(reg[blk * 4 + 0], w) >> sh) & 0xffffu;
        const uint32_t e1 = (word_of(reg[blk * 4 + 1], w) >> sh) & 0xffffu;
        const uint32_t e2 = (word_of(reg[blk * 4 + 2], w) >> sh) & 0xffffu;
        const uint32_t e3 = (word_of(reg[blk * 4 + 3], w) >> sh) & 0xffffu;
        piece.x = e0 | (e1 << 16);
        piece.y = e2 | (e3 << 16);
        if constexpr (kSum)
          colsum[v] += (bf16_to_f32(e0) + bf16_to_f32(e1)) + (bf16_to_f32(e2) + bf16_to_f32(e3));
      } else {
        piece.x = word_of(reg[blk * 2 + 0], v);
        piece.y = word_of(reg[blk * 2 + 1], v);
        if constexpr (kSum) colsum[v] += __uint_as_float(piece.x) + __uint_as_float(piece.y);
      }
      *reinterpret_cast<uint2*>(lds + (cb * G::VEC + v) * kRowBytes + kb * G::TK * sizeof(T)) =
          piece;
    }
  }
}

template <typename T>
__device__ __forceinline__ void compute_step(const char* As, const char* Bs, f32x16_t (&acc)[2][2]) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int lr = lane & 31, lh = lane >> 5;
  const char* a_base = As + (wm * 64 + lr) * kRowBytes + lh * 16;
  const char* b_base = Bs + (wn * 64 + lr) * kRowBytes + lh * 16;
#pragma unroll
  for (int rs = 0; rs < 4; ++rs) {
    const uint4 a0 = *reinterpret_cast<const uint4*>(a_base + rs * 32);
    const uint4 a1 = *reinterpret_cast<const uint4*>(a_base + 32 * kRowBytes + rs * 32);
    const uint4 b0 = *reinterpret_cast<const uint4*>(b_base + rs * 32);
    const uint4 b1 = *reinterpret_cast<const uint4*>(b_base + 32 * kRowBytes + rs * 32);
    mma(acc[0][0], a0, b0, T());
    mma(acc[0][1], a0, b1, T());
    mma(acc[1][0], a1, b0, T());
    mma(acc[1][1], a1, b1, T());
  }
}

// Local row / column of C held by accumulator element e of block (mi, ni).
__device__ __forceinline__ int acc_row(int mi, int e) {
  const int lane = threadIdx.x & 63;
  const int wm = (threadIdx.x >> 6) >> 1;
  return wm * 64 + mi * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
}
__device__ __forceinline__ int acc_col(int ni) {
  const int lane = threadIdx.x & 63;
  const int wn = (threadIdx.x >> 6) & 1;
  return wn * 64 + ni * 32 + (lane & 31);
}

template <typename T, int MODE>
__global__ __launch_bounds__(kThreads, 2) void star_gemm_kernel(const GemmParams p) {
  constexpr int BK = Traits<T>::BK;
  __shared__ __attribute__((aligned(16))) char smem[kSmemBytes];
  __shared__ int32_t rows_s[BM];
  __shared__ int32_t units_s[kMaxQGroups];
  __shared__ int32_t pfx_s[kMaxQGroups + 1];

  auto As = [&](int buf) { return smem + buf * kTileBytes; };
  auto Bs = [&](int buf) { return smem + (2 + buf) * kTileBytes; };
  const T* __restrict__ Ag = static_cast<const T*>(p.A);
  const T* __restrict__ Bg = static_cast<const T*>(p.B);
  const int q = p.q;

  // row units per class: row tiles of I_i (FWD, BWD_DATA) or row tiles of
  // input group g times the split count (BWD_WEIGHT)
  for (int i = threadIdx.x; i < q; i += kThreads) {
    if constexpr (MODE == kModeBwdWeight) {
      units_s[i] = (p.MTp[i + 1] - p.MTp[i]) * p.nsplit;
    } else {
      const int32_t mi = p.offsets[i + 1] - p.offsets[i];
      units_s[i] = (mi + BM - 1) / BM;
    }
  }

  const int xcd = blockIdx.x & 7;
  const int slot0 = blockIdx.x >> 3;
  const int slot_stride = gridDim.x >> 3;

  for (int pass = 0; pass < 2; ++pass) {
    const int sel = sel_for(MODE, p.law, pass);
    __syncthreads();
    if (threadIdx.x == 0) {
      int32_t run = 0;
      for (int i = 0; i < q; ++i) {
        pfx_s[i] = run;
        run += units_s[i] * ncols_sel(p, sel, i);
      }
      pfx_s[q] = run;
    }
    __syncthreads();
    const int32_t total = pfx_s[q];
    const int32_t chunk = (total + 7) >> 3;

    for (int32_t slot = slot0; slot < chunk; slot += slot_stride) {
      const int32_t logical = xcd * chunk + slot;
      if (logical >= total) break;
      int cls = 0;
      while (logical >= pfx_s[cls + 1]) ++cls;
      const int32_t u = logical - pfx_s[cls];
      const int32_t ru = u % units_s[cls];
      const int ct = col_tile_global(p, sel, cls, u / units_s[cls]);
      int cg = 0;
      while (ct >= p.NTp[cg + 1]) ++cg;
      const int nt = ct - p.NTp[cg];

      // ---- tile geometry -------------------------------------------------
      int32_t cstart, cend;          // columns of C (global index space)
      int32_t seg0_lo = 0, seg0_hi = 0, seg1_lo = 0, seg1_hi = 0;  // K ranges
      int32_t rstart = 0, rend = 0;  // BWD_WEIGHT: rows of C (kk)
      int32_t split = 0, mt;
      bool do_dbias = false;
      if constexpr (MODE == kModeFwd) {
        mt = ru;
        cstart = p.R[cg] + nt * BN;
        cend = p.R[cg + 1];
        if (p.law == 1) {
          seg0_lo = 0; seg0_hi = p.K;
        } else {
          seg0_lo = p.S[cg]; seg0_hi = p.S[cg + 1];
          if (cg != cls) { seg1_lo = p.S[cls]; seg1_hi = p.S[cls + 1]; }
        }
      } else if constexpr (MODE == kModeBwdData) {
        mt = ru;
        cstart = p.S[cg] + nt * BN;
        cend = p.S[cg + 1];
        if (p.law == 1 || cg == cls) {
          seg0_lo = 0; seg0_hi = p.N;
        } else {
          seg0_lo = p.R[cg]; seg0_hi = p.R[cg + 1];
        }
      } else {
        mt = ru / p.nsplit;
        split = ru % p.nsplit;
        cstart = p.R[cg] + nt * BN;
        cend = p.R[cg + 1];
        rstart = p.S[cls] + mt * BM;
        rend = p.S[cls + 1];
        int32_t lo, hi;
        if (p.law == 0 && cg != cls) {
          lo = p.offsets[cls]; hi = p.offsets[cls + 1];
        } else {
          lo = 0; hi = p.offsets[q];
        }
        const int32_t len = hi - lo;
        const int32_t cs = (len + p.nsplit - 1) / p.nsplit;
        seg0_lo = min(hi, lo + split * cs);
        seg0_hi = min(hi, seg0_lo + cs);
        do_dbias = (p.dbias != nullptr) && (cg == cls) && (mt == 0);
      }
      const int32_t n0 = (seg0_hi - seg0_lo + BK - 1) / BK;
      const int32_t n1 = (seg1_hi - seg1_lo + BK - 1) / BK;
      const int32_t nsteps = n0 + n1;

      __syncthreads();  // previous tile is done with rows_s and LDS
      if constexpr (MODE != kModeBwdWeight) {
        const int32_t pos0 = p.offsets[cls] + mt * BM;
        const int32_t nrows = min(BM, p.offsets[cls + 1] - pos0);
        if (threadIdx.x < BM) rows_s[threadIdx.x] = threadIdx.x < nrows ? p.perm[pos0 + threadIdx.x] : -1;
      }
      __syncthreads();

      int32_t arow[4];
      int32_t brow[4];
      if constexpr (MODE != kModeBwdWeight) {
#pragma unroll
        for (int u = 0; u < 4; ++u) arow[u] = rows_s[(threadIdx.x >> 3) + 32 * u];
      }
      if constexpr (MODE == kModeBwdData) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int32_t kk = cstart + (threadIdx.x >> 3) + 32 * u;
          brow[u] = kk < cend ? kk : -1;
        }
      }

      float colsum[8];
#pragma unroll
      for (int v = 0; v < 8; ++v) colsum[v] = 0.f;

      auto step_range = [&](int32_t s, int32_t& k0, int32_t& kend) {
        if (s < n0) { k0 = seg0_lo + s * BK; kend = seg0_hi; }
        else { k0 = seg1_lo + (s - n0) * BK; kend = seg1_hi; }
      };

      uint4 ra[4], rb[4];
      auto load_stage = [&](int32_t s) {
        int32_t k0, kend;
        step_range(s, k0, kend);
        if constexpr (MODE == kModeFwd) {
          load_k<T>(ra, Ag, p.K, arow, k0, kend);
          load_t<T>(rb, Bg, p.N, k0, cstart, cend,
                    [&](int32_t k) { return k < kend ? k : -1; });
        } else if constexpr (MODE == kModeBwdData) {
          load_k<T>(ra, Ag, p.N, arow, k0, kend);
          load_k<T>(rb, Bg, p.N, brow, k0, kend);
        } else {
          const int32_t* __restrict__ perm = p.perm;
          auto srow = [&](int32_t k) { return k < kend ? perm[k] : -1; };
          load_t<T>(ra, Ag, p.K, k0, rstart, rend, srow);
          load_t<T>(rb, Bg, p.N, k0, cstart, cend, srow);
        }
      };
      auto store_stage = [&](int buf) {
        if constexpr (MODE == kModeFwd) {
          store_k(As(buf), ra);
          store_t<T, false>(Bs(buf), rb, colsum);
        } else if constexpr (MODE == kModeBwdData) {
          store_k(As(buf), ra);
          store_k(Bs(buf), rb);
        } else {
          store_t<T, false>(As(buf), ra, colsum);
          if (do_dbias) store_t<T, true>(Bs(buf), rb, colsum);
          else store_t<T, false>(Bs(buf), rb, colsum);
        }
      };

      f32x16_t acc[2][2];
#pragma unroll
      for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 2; ++ni)
#pragma unroll
          for (int e = 0; e < 16; ++e) acc[mi][ni][e] = 0.f;

      if (nsteps > 0) {
        load_stage(0);
        store_stage(0);
        __syncthreads();
        for (int32_t s = 0; s < nsteps; ++s) {
          if (s + 1 < nsteps) load_stage(s + 1);
          compute_step<T>(As(s & 1), Bs(s & 1), acc);
          if (s + 1 < nsteps) store_stage((s + 1) & 1);
          __syncthreads();
        }
      }

      // ---- epilogue --------------------------------------------------------
      if constexpr (MODE == kModeFwd) {
#pragma unroll
        for (int ni = 0; ni < 2; ++ni) {
          const int32_t gcol = cstart + acc_col(ni);
          if (gcol >= cend) continue;
          const float bv = p.bias ? p.bias[gcol] : 0.f;
#pragma unroll
          for (int mi = 0; mi < 2; ++mi)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
              const int32_t grow = rows_s[acc_row(mi, e)];
              if (grow < 0) continue;
              const float z = acc[mi][ni][e] + bv;
              const int64_t idx = static_cast<int64_t>(grow) * p.N + gcol;
              if (p.Z) store_out(p.Z, p.ydtype, idx, z);
              store_out(p.Y, p.ydtype, idx, act_fwd(p.act, z));
            }
        }
      } else if constexpr (MODE == kModeBwdData) {
#pragma unroll
        for (int ni = 0; ni < 2; ++ni) {
          const int32_t gcol = cstart + acc_col(ni);
          if (gcol >= cend) continue;
#pragma unroll
          for (int mi = 0; mi < 2; ++mi)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
              const int32_t grow = rows_s[acc_row(mi, e)];
              if (grow < 0) continue;
              const int64_t idx = static_cast<int64_t>(grow) * p.K + gcol;
              float v = acc[mi][ni][e];
              if (p.Zprev) v *= act_grad(p.act, load_in(p.Zprev, p.elem == 0 ? 0 : 1, idx));
              store_out(p.Y, p.ydtype, idx, v);
            }
        }
      } else {
        float* out = p.nsplit > 1 ? p.partial + static_cast<int64_t>(split) * p.K * p.N : p.dW;
#pragma unroll
        for (int ni = 0; ni < 2; ++ni) {
          const int32_t gcol = cstart + acc_col(ni);
          if (gcol >= cend) continue;
#pragma unroll
          for (int mi = 0; mi < 2; ++mi)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
              const int32_t grow = rstart + acc_row(mi, e);
              if (grow >= rend) continue;
              out[static_cast<int64_t>(grow) * p.N + gcol] = acc[mi][ni][e];
            }
        }
        if (do_dbias) {
          // column sums of the staged dY: thread t holds column chunk
          // t % CB; reduce over the threads sharing it through LDS.
          using G = TGeom<T>;
          constexpr int kSlots = kThreads / G::CB;
          float* red = reinterpret_cast<float*>(smem);
          const int cb = threadIdx.x % G::CB;
          const int slotr = threadIdx.x / G::CB;
#pragma unroll
          for (int v = 0; v < G::VEC; ++v) red[slotr * BN + cb * G::VEC + v] = colsum[v];
          __syncthreads();
          if (threadIdx.x < BN) {
            float sum = 0.f;
            for (int sl = 0; sl < kSlots; ++sl) sum += red[sl * BN + threadIdx.x];
            const int32_t gcol = cstart + threadIdx.x;
            if (gcol < cend) {
              if (p.nsplit > 1) p.dbias_part[static_cast<int64_t>(split) * p.N + gcol] = sum;
              else p.dbias[gcol] = sum;
            }
          }
        }
      }
    }
  }
}

__global__ void split_reduce_kernel(const float* __restrict__ part, int nsplit, int64_t n,
                                    float* __restrict__ out) {
  const int64_t n4 = n >> 2;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n4;
       i += (int64_t)gridDim.x * blockDim.x) {
    float4 acc = reinterpret_cast<const float4*>(part)[i];
    for (int s = 1; s < nsplit; ++s) {
      const float4 v = reinterpret_cast<const float4*>(part + static_cast<int64_t>(s) * n)[i];
      acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
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

template <typename T, int MODE>
hipError_t launch_typed(const GemmParams& p, int grid, hipStream_t stream) {
  hipLaunchKernelGGL((star_gemm_kernel<T, MODE>), dim3(grid), dim3(kThreads), 0, stream, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm(int mode, const GemmParams& p, int grid, hipStream_t stream) {
  if (p.elem == 1) {
    if (mode == kModeFwd) return launch_typed<uint16_t, kModeFwd>(p, grid, stream);
    if (mode == kModeBwdData) return launch_typed<uint16_t, kModeBwdData>(p, grid, stream);
    return launch_typed<uint16_t, kModeBwdWeight>(p, grid, stream);
  }
  if (mode == kModeFwd) return launch_typed<float, kModeFwd>(p, grid, stream);
  if (mode == kModeBwdData) return launch_typed<float, kModeBwdData>(p, grid, stream);
  return launch_typed<float, kModeBwdWeight>(p, grid, stream);
}

hipError_t launch_fill_zero(float* dst, int64_t n, hipStream_t stream) {
  const int blocks = static_cast<int>(std::min<int64_t>(1024, (n + 255) / 256 + 1));
  hipLaunchKernelGGL(fill_zero_kernel, dim3(blocks), dim3(256), 0, stream, dst, n);
  return hipGetLastError();
}

hipError_t launch_split_reduce(const GemmParams& p, hipStream_t stream) {
  const int64_t nKN = static_cast<int64_t>(p.K) * p.N;
  int blocks = static_cast<int>(std::min<int64_t>(2048, (nKN / 4 + 255) / 256 + 1));
  hipLaunchKernelGGL(split_reduce_kernel, dim3(blocks), dim3(256), 0, stream, p.partial,
                     p.nsplit, nKN, p.dW);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.dbias == nullptr) return e;
  hipLaunchKernelGGL(split_reduce_kernel, dim3(8), dim3(256), 0, stream, p.dbias_part, p.nsplit,
                     static_cast<int64_t>(p.N), p.dbias);
  return hipGetLastError();
}

}  // namespace starq
