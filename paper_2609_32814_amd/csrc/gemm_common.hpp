// Pieces shared by the grouped GEMM kernels: tile enumeration, MFMA
// wrappers and 4-wide output stores.
#pragma once

#include "common.hpp"
#include "kernels.hpp"

namespace starq {
namespace gemm {

constexpr int BM = kTileM;  // 256
constexpr int THREADS = 256;

template <typename T> struct Tr;
template <> struct Tr<float> {
  static constexpr int VEC = 4;  // elements per 16-byte kpack
  static constexpr int BK = 32;  // K per step: 8 kpacks
};
template <> struct Tr<uint16_t> {
  static constexpr int VEC = 8;
  static constexpr int BK = 64;
};

template <int WN> struct Geo {
  static constexpr int BN = 64 * WN;
  static constexpr int A_BYTES = 8 * BM * 16;
  static constexpr int B_BYTES = 8 * BN * 16;
  static constexpr int STAGE = A_BYTES + B_BYTES;
  static constexpr int SMEM = 2 * STAGE;
};

__device__ __forceinline__ int swz(int row, int kp) { return row ^ (((row >> 3) ^ kp) & 7); }

template <int ROWS>
__device__ __forceinline__ int unit_off(int kp, int row) {
  return (kp * ROWS + swz(row, kp)) * 16;
}

__device__ __forceinline__ uint32_t word_of(const uint4& r, int w) {
  return w == 0 ? r.x : (w == 1 ? r.y : (w == 2 ? r.z : r.w));
}

enum Sel : int { kSelNone = 0, kSelOnly = 1, kSelExcept = 2, kSelAll = 3, kSelTensor = 4, kSelGraph = 10 };

// Law 2, the tensor power of the two-group law (q = 2^L): input group k is
// in B(i, j) when every bit of k equals that bit of i or of j.
__device__ __forceinline__ bool tensor_in_support(int i, int j, int k) { return ((k ^ i) & (k ^ j)) == 0; }

// Law 2: bit x set when x is in the contraction of a tile of class i (a row
// type; for the weight gradient an input group) and C-column group j:
//  forward: input groups x in B(i, j);
//  activation gradient (C columns are input group j): output groups x with
//  j in B(i, x);
//  weight gradient (C rows input group i, columns output group j): row
//  types x with i in B(x, j).
__device__ __forceinline__ uint32_t tensor_mask(int mode, int q, int i, int j) {
  uint32_t m = 0;
  for (int x = 0; x < q; ++x) {
    const bool in = mode == kModeFwd ? tensor_in_support(i, j, x)
                                     : (mode == kModeBwdData ? tensor_in_support(i, x, j) : tensor_in_support(x, j, i));
    if (in) m |= 1u << x;
  }
  return m;
}
// maximal runs of consecutive set bits (each run is one contiguous range)
__device__ __forceinline__ int mask_runs(uint32_t m) { return __popc(m & ~(m << 1)); }
// the first two runs: [lo0, hi0) and [lo1, hi1) (empty when absent)
__device__ __forceinline__ void mask_ranges(uint32_t m, int& lo0, int& hi0, int& lo1, int& hi1) {
  lo0 = hi0 = lo1 = hi1 = 0;
  if (!m) return;
  lo0 = __builtin_ctz(m);
  hi0 = lo0 + __builtin_ctz(~(m >> lo0));
  const uint32_t rest = hi0 >= 32 ? 0u : (m & ~((1u << hi0) - 1u));
  if (!rest) return;
  lo1 = __builtin_ctz(rest);
  hi1 = lo1 + __builtin_ctz(~(rest >> lo1));
}

// Law 3, the graph algebra Q_G (bit j of p.adj[i] marks the edge i -> j): a
// type-i row's slots are its vertex slot i and the edge slots of its
// out-edges, so B(i,i) = {i}, B(i,j) = {i, j} for an edge i -> j and B(i,j)
// is empty for a non-edge.  Bit x set when x is in the contraction of a tile
// of class i and C-column group j, as for tensor_mask.
__device__ __forceinline__ uint64_t graph_mask(const GemmParams& p, int mode, int i, int j) {
  const uint64_t bi = 1ull << i, bj = 1ull << j;
  const bool edge = (p.adj[i] >> j) & 1ull;
  if (mode == kModeFwd) return j == i ? bi : (edge ? (bi | bj) : 0ull);
  if (mode == kModeBwdData) return j == i ? (bi | p.adj[i]) : (edge ? bj : 0ull);
  // weight gradient (C rows input group i, columns output group j): the row
  // types x whose B(x, j) holds i: for i = j, j itself and every x with an
  // edge x -> j; for i != j, i itself if it has the edge i -> j
  return i == j ? (bj | p.adj_in[j]) : (edge ? bi : 0ull);
}
// law 3: pass 0 holds the tiles that contract over two or more groups, pass 1
// those over one; tiles over none are in no pass (their outputs are not
// slots: launch_graph_fill writes them) except in the weight gradient,
// whose pass 1 holds them (they are written as zeros)
__device__ __forceinline__ bool graph_in_pass(const GemmParams& p, int sel, int i, int j) {
  const int mode = (sel - kSelGraph) >> 1, pass = (sel - kSelGraph) & 1;
  const int n = __popcll(graph_mask(p, mode, i, j));
  return pass == 0 ? n >= 2 : (n == 1 || (n == 0 && mode == kModeBwdWeight));
}

// Law 3: the contraction of a tile is the concatenation, in group order, of
// the ranges [bound(x), bound(x + 1)) of the groups x in `mask` (bound: input
// group starts, output group starts or type offsets), cut to positions
// [c0, c1) of that concatenation; a K step never straddles two groups.
template <int BK, typename BF>
__device__ __forceinline__ int32_t graph_steps(uint64_t mask, BF bound, int32_t c0, int32_t c1) {
  int32_t steps = 0, cum = 0;
  while (mask) {
    const int x = __builtin_ctzll(mask);
    mask &= mask - 1;
    const int32_t lo = bound(x), len = bound(x + 1) - lo;
    const int32_t a = max(cum, c0), b = min(cum + len, c1);
    if (b > a) steps += (b - a + BK - 1) / BK;
    cum += len;
  }
  return steps;
}
template <int BK, typename BF>
__device__ __forceinline__ void graph_step_range(uint64_t mask, BF bound, int32_t c0, int32_t c1, int32_t st,
                                                 int32_t& lo_out, int32_t& hi_out) {
  int32_t cum = 0;
  lo_out = hi_out = 0;
  while (mask) {
    const int x = __builtin_ctzll(mask);
    mask &= mask - 1;
    const int32_t lo = bound(x), len = bound(x + 1) - lo;
    const int32_t a = max(cum, c0), b = min(cum + len, c1);
    if (b > a) {
      const int32_t n = (b - a + BK - 1) / BK;
      if (st < n) {
        lo_out = lo + (a - cum) + st * BK;
        hi_out = lo + (b - cum);
        return;
      }
      st -= n;
    }
    cum += len;
  }
}

// A pass selects, per class, the C-column groups of its tiles: the star
// law puts the tiles with two K segments first, the dense law has one pass;
// law 2 puts the tiles that contract over more than half of the groups
// first, with the mode folded into the selector.
__device__ __forceinline__ int sel_for(int mode, int law, int pass) {
  if (law == 1) return pass == 0 ? kSelAll : kSelNone;
  if (law == 3) return kSelGraph + 2 * mode + pass;
  if (law == 2) return kSelTensor + 2 * mode + pass;
  if (mode == kModeFwd) return pass == 0 ? kSelExcept : kSelOnly;
  return pass == 0 ? kSelOnly : kSelExcept;  // BWD_DATA and BWD_WEIGHT
}
// law 2: is column group j of class i in the selector's pass?  Pass 0
// holds the tiles whose contraction spans more than half of the groups (the
// longest), pass 1 the rest, so that long tiles start first.
__device__ __forceinline__ bool tensor_in_pass(const GemmParams& p, int sel, int i, int j) {
  const int mode = (sel - kSelTensor) >> 1, pass = (sel - kSelTensor) & 1;
  const bool wide = 2 * static_cast<int>(__popc(tensor_mask(mode, p.q, i, j))) > p.q;
  return pass == 0 ? wide : !wide;
}

__device__ __forceinline__ int ncols_sel(const GemmParams& p, int sel, int i) {
  const int nti = p.NTp[i + 1] - p.NTp[i];
  const int nt = p.NTp[p.q];
  if (sel >= kSelGraph) {
    int n = 0;
    for (int j = 0; j < p.q; ++j)
      if (graph_in_pass(p, sel, i, j)) n += p.NTp[j + 1] - p.NTp[j];
    return n;
  }
  if (sel >= kSelTensor) {
    int n = 0;
    for (int j = 0; j < p.q; ++j)
      if (tensor_in_pass(p, sel, i, j)) n += p.NTp[j + 1] - p.NTp[j];
    return n;
  }
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
  if (sel >= kSelGraph) {
    for (int j = 0; j < p.q; ++j) {
      if (!graph_in_pass(p, sel, i, j)) continue;
      const int ntj = p.NTp[j + 1] - p.NTp[j];
      if (c < ntj) return p.NTp[j] + c;
      c -= ntj;
    }
    return p.NTp[p.q];  // not reached: c < ncols_sel
  }
  if (sel >= kSelTensor) {
    // the c-th column tile over the pass's groups, in group order
    for (int j = 0; j < p.q; ++j) {
      if (!tensor_in_pass(p, sel, i, j)) continue;
      const int ntj = p.NTp[j + 1] - p.NTp[j];
      if (c < ntj) return p.NTp[j] + c;
      c -= ntj;
    }
    return p.NTp[p.q];  // not reached: c < ncols_sel
  }
  return c;
}

// D += A B with the operands of the C^T block: a = B-tile fragment (rows of
// D are columns of C), b = A-tile fragment (columns of D are rows of C).
__device__ __forceinline__ void mma(f32x16_t& acc, const uint4& a, const uint4& b, uint16_t) {
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                __builtin_bit_cast(bf16x8_t, b), acc, 0, 0, 0);
}
__device__ __forceinline__ void mma(f32x16_t& acc, const uint4& a, const uint4& b, float) {
  // lane half h supplies K element 4 kp + j of instruction j; both operands
  // use the same assignment, so the products pair up.
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
}

// 4 consecutive values of a row of an fp32 or bf16 matrix
__device__ __forceinline__ void store4(void* base, int dtype, int64_t idx, const float (&v)[4]) {
  if (dtype == 0) {
    *reinterpret_cast<float4*>(static_cast<float*>(base) + idx) = make_float4(v[0], v[1], v[2], v[3]);
  } else {
    uint2 w;
    w.x = static_cast<uint32_t>(f32_to_bf16(v[0])) | (static_cast<uint32_t>(f32_to_bf16(v[1])) << 16);
    w.y = static_cast<uint32_t>(f32_to_bf16(v[2])) | (static_cast<uint32_t>(f32_to_bf16(v[3])) << 16);
    *reinterpret_cast<uint2*>(static_cast<uint16_t*>(base) + idx) = w;
  }
}

__device__ __forceinline__ void load4(const void* base, int dtype, int64_t idx, float (&v)[4]) {
  if (dtype == 0) {
    const float4 f = *reinterpret_cast<const float4*>(static_cast<const float*>(base) + idx);
    v[0] = f.x; v[1] = f.y; v[2] = f.z; v[3] = f.w;
  } else {
    const uint2 w = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(base) + idx);
    v[0] = bf16_to_f32(w.x & 0xffffu); v[1] = bf16_to_f32(w.x >> 16);
    v[2] = bf16_to_f32(w.y & 0xffffu); v[3] = bf16_to_f32(w.y >> 16);
  }
}

// One 16-byte load that reads zeros when `ok` is false.  The address is
// clamped to the (always valid) first element instead of branching.
template <typename T>
__device__ __forceinline__ uint4 load16(const T* __restrict__ src, int64_t off, bool ok) {
  const uint4 v = *reinterpret_cast<const uint4*>(src + (ok ? off : 0));
  return ok ? v : make_uint4(0, 0, 0, 0);
}

// ---- tile iteration ----------------------------------------------------------

struct Tile {
  int32_t cls, cg, mt, split;
  int32_t cstart, cend;                          // columns of C
  int32_t rstart, rend;                          // BWD_WEIGHT: rows of C
  int32_t seg0_lo, seg0_hi, seg1_lo, seg1_hi;    // K ranges
  int32_t n0, nsteps;                            // K steps in segment 0, in total
  int32_t pos0, nrows;                           // FWD/BWD_DATA: rows in perm
  int32_t do_dbias;
};

// `offs` holds the q + 1 type offsets of the plan (global memory or an LDS
// copy).  Forward and activation gradient: row tiles are `bm` rows (BM, or
// BM / 2 for the half-height tiles that balance a short last round).
template <int MODE, int LAW, int BN, int BK>
__device__ __forceinline__ Tile make_tile(const GemmParams& p, int sel, int cls, int32_t u,
                                          int32_t units, const int32_t* offs, int bm = BM) {
  Tile t;
  // Forward and activation gradient: column tiles vary fastest, so that the
  // tiles of one XCD chunk cover a few row tiles across all their column
  // tiles (their rows stay in that XCD's L2 while the weights stream).
  // Weight gradient: row-tile x split units vary fastest.
  int32_t ru, cidx;
  if constexpr (MODE == kModeBwdWeight) {
    ru = u % units;
    cidx = u / units;
  } else {
    const int32_t nc = ncols_sel(p, sel, cls);
    ru = u / nc;
    cidx = u % nc;
  }
  const int ct = col_tile_global(p, sel, cls, cidx);
  int cg = 0;
  while (cg + 1 < p.q && ct >= p.NTp[cg + 1]) ++cg;
  const int nt = ct - p.NTp[cg];
  t.cls = cls;
  t.cg = cg;
  t.seg1_lo = t.seg1_hi = 0;
  t.rstart = t.rend = 0;
  t.split = 0;
  t.do_dbias = 0;
  t.pos0 = t.nrows = 0;
  if constexpr (MODE == kModeFwd) {
    t.mt = ru;
    t.cstart = p.R[cg] + nt * BN;
    t.cend = p.R[cg + 1];
    if (LAW == 1 || LAW == 3) {
      t.seg0_lo = 0; t.seg0_hi = p.K;
    } else if (LAW == 2) {
      int a0, a1, b0, b1;
      mask_ranges(tensor_mask(kModeFwd, p.q, cls, cg), a0, a1, b0, b1);
      t.seg0_lo = p.S[a0]; t.seg0_hi = p.S[a1];
      t.seg1_lo = p.S[b0]; t.seg1_hi = p.S[b1];
    } else {
      t.seg0_lo = p.S[cg]; t.seg0_hi = p.S[cg + 1];
      if (cg != cls) { t.seg1_lo = p.S[cls]; t.seg1_hi = p.S[cls + 1]; }
    }
  } else if constexpr (MODE == kModeBwdData) {
    t.mt = ru;
    t.cstart = p.S[cg] + nt * BN;
    t.cend = p.S[cg + 1];
    if (LAW == 2) {
      int a0, a1, b0, b1;
      mask_ranges(tensor_mask(kModeBwdData, p.q, cls, cg), a0, a1, b0, b1);
      t.seg0_lo = p.R[a0]; t.seg0_hi = p.R[a1];
      t.seg1_lo = p.R[b0]; t.seg1_hi = p.R[b1];
    } else if (LAW == 1 || LAW == 3 || cg == cls) {
      t.seg0_lo = 0; t.seg0_hi = p.N;
    } else {
      t.seg0_lo = p.R[cg]; t.seg0_hi = p.R[cg + 1];
    }
  } else {
    t.mt = ru / p.nsplit;
    t.split = ru % p.nsplit;
    t.cstart = p.R[cg] + nt * BN;
    t.cend = p.R[cg + 1];
    t.rstart = p.S[cls] + t.mt * bm;
    t.rend = p.S[cls + 1];
    // the type-sorted positions this tile contracts over: one or two
    // ranges, cut into nsplit chunks of their concatenation
    int32_t a0, a1, b0 = 0, b1 = 0;
    if (LAW == 2) {
      int ta0, ta1, tb0, tb1;
      mask_ranges(tensor_mask(kModeBwdWeight, p.q, cls, cg), ta0, ta1, tb0, tb1);
      a0 = offs[ta0]; a1 = offs[ta1];
      b0 = offs[tb0]; b1 = offs[tb1];
    } else if (LAW == 0 && cg != cls) {
      a0 = offs[cls]; a1 = offs[cls + 1];
    } else if (LAW == 3) {
      a0 = a1 = 0;  // set below from the graph mask
    } else {
      a0 = 0; a1 = offs[p.q];
    }
    const int32_t len0 = a1 - a0, len = len0 + (b1 - b0);
    const int32_t cs = (len + p.nsplit - 1) / p.nsplit;
    const int32_t c0 = min(len, t.split * cs), c1 = min(len, c0 + cs);
    t.seg0_lo = a0 + min(c0, len0);
    t.seg0_hi = a0 + min(c1, len0);
    t.seg1_lo = b0 + max(c0 - len0, 0);
    t.seg1_hi = b0 + max(c1 - len0, 0);
    t.do_dbias = (p.dbias != nullptr) && (cg == cls) && (t.mt == 0);
  }
  if constexpr (MODE != kModeBwdWeight) {
    t.pos0 = offs[cls] + t.mt * bm;
    t.nrows = min(bm, offs[cls + 1] - t.pos0);
  }
  if constexpr (LAW == 3) {
    // the graph law: seg0 holds the contraction's group mask, seg1 the
    // positions [c0, c1) of its concatenated ranges this tile covers (all
    // of them, or the split's chunk for the weight gradient)
    const uint64_t m = graph_mask(p, MODE, cls, cg);
    int32_t total = 0, c0 = 0, c1 = 0;
    auto count = [&](auto bound) {
      for (uint64_t r = m; r; r &= r - 1) {
        const int x = __builtin_ctzll(r);
        total += bound(x + 1) - bound(x);
      }
      if (MODE == kModeBwdWeight) {
        const int32_t cs = (total + p.nsplit - 1) / p.nsplit;
        c0 = min(total, t.split * cs);
        c1 = min(total, c0 + cs);
      } else {
        c1 = total;
      }
      t.nsteps = graph_steps<BK>(m, bound, c0, c1);
    };
    if constexpr (MODE == kModeFwd) count([&](int x) { return p.S[x]; });
    else if constexpr (MODE == kModeBwdData) count([&](int x) { return p.R[x]; });
    else count([&](int x) { return offs[x]; });
    t.seg0_lo = static_cast<int32_t>(static_cast<uint32_t>(m));
    t.seg0_hi = static_cast<int32_t>(static_cast<uint32_t>(m >> 32));
    t.seg1_lo = c0;
    t.seg1_hi = c1;
    t.n0 = 0;
    // the bias gradient sums every row; the graph law's diagonal blocks do
    // not contract over all of them, so it is summed apart
    t.do_dbias = 0;
  } else {
    t.n0 = (t.seg0_hi - t.seg0_lo + BK - 1) / BK;
    t.nsteps = t.n0 + (t.seg1_hi - t.seg1_lo + BK - 1) / BK;
  }
  // every field is uniform over the workgroup: keep it in scalar registers
  int32_t* f = reinterpret_cast<int32_t*>(&t);
#pragma unroll
  for (int k = 0; k < static_cast<int>(sizeof(Tile) / sizeof(int32_t)); ++k)
    f[k] = __builtin_amdgcn_readfirstlane(f[k]);
  return t;
}

// K range of step st of tile t: [lo, ...) with the end of its segment in hi
// (offs: the type offsets, for the weight gradient's positions).
template <int MODE, int LAW, int BK>
__device__ __forceinline__ void step_range(const GemmParams& p, const Tile& t, const int32_t* offs, int32_t st,
                                           int32_t& lo, int32_t& hi) {
  if constexpr (LAW == 3) {
    const uint64_t m = static_cast<uint64_t>(static_cast<uint32_t>(t.seg0_lo)) |
                       (static_cast<uint64_t>(static_cast<uint32_t>(t.seg0_hi)) << 32);
    if constexpr (MODE == kModeFwd)
      graph_step_range<BK>(m, [&](int x) { return p.S[x]; }, t.seg1_lo, t.seg1_hi, st, lo, hi);
    else if constexpr (MODE == kModeBwdData)
      graph_step_range<BK>(m, [&](int x) { return p.R[x]; }, t.seg1_lo, t.seg1_hi, st, lo, hi);
    else
      graph_step_range<BK>(m, [&](int x) { return offs[x]; }, t.seg1_lo, t.seg1_hi, st, lo, hi);
  } else if (st < t.n0) {
    lo = t.seg0_lo + st * BK;
    hi = t.seg0_hi;
  } else {
    lo = t.seg1_lo + (st - t.n0) * BK;
    hi = t.seg1_hi;
  }
}

}  // namespace gemm
}  // namespace starq
