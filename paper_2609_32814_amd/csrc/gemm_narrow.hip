// Forward product for many small groups (§"Kernels"; §"Kernel Scaling on
// Transformer Shapes"): when each row type has few rows (M / q well below a
// 256-row tile) or the groups are narrow, the 256 x 256 tiles of the
// persistent GEMM are mostly empty.  Here a tile is 64 rows of one type
// (rows taken in type order through the plan) x 128 columns of one output
// group, the contraction is the concatenation of the input groups in the
// law's B(i, j) (at most two contiguous K ranges for every law; it runs in
// 64-deep K steps that may span both ranges, and the last one is zero-filled
// past its end), and a workgroup of 4 wavefronts (2 x 2, each 32 rows
// x 64 columns: two v_mfma_f32_32x32x16_bf16 blocks) computes it with both
// operands staged in LDS by direct global-to-LDS copies.  Workgroups are
// persistent: each walks its tiles as one stream of K steps whose copies run
// two steps ahead across tile boundaries (each tile has few steps), with the
// rows of the next tiles fetched while earlier tiles compute.
// Bias, activation, an optional pre-activation store and the bf16/fp32
// output follow in the epilogue.
//
// Work order: workgroup w runs on XCD w mod 8; each XCD owns an eighth of
// the row blocks (or of the column tiles, when there are fewer than 8 row
// blocks) and sweeps the column tiles band by band of its row blocks, so a
// weight tile is fetched once per band and the band's rows stay in L2.
//
// The paper's second schedule (the diagonal maps over all rows, then the
// type-dependent maps) serves the same regime; here both products of a
// tile are accumulated in registers before one output store.
#include <algorithm>
#include <type_traits>

#include "gemm_common.hpp"

namespace starq {

namespace {

using namespace gemm;

constexpr int kNThreads = 256;
constexpr int kNRows = 64;                 // rows per tile
constexpr int kNCols = 128;                // columns per tile
constexpr int kNK = 64;                    // K per step
constexpr int kA = kNRows * kNK * 2;       // 8 KB
constexpr int kB = kNK * kNCols * 2;       // 16 KB
constexpr int kStage = kA + kB;
constexpr int kNStages = 3;                // copies run two K steps ahead
constexpr int kNSmem = kNStages * kStage;  // 72 KB: two workgroups per CU
constexpr int kSlots = 5;                  // tiles described in LDS (the consumer's and 4 ahead)

typedef short v4i16_t __attribute__((ext_vector_type(4)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
#define STARQ_LDS __attribute__((address_space(3)))

// source of the copies that must land as zeros
__device__ __attribute__((aligned(256))) uint32_t g_narrow_zero[256];
// Where the epilogue's lanes without an output element store: every lane
// stores each of its output blocks, so the number of stores in flight is
// known.  A lane's sink covers one row of its blocks (at most 240 bytes);
// kSinkSets sets of 64 lanes spread the writes over workgroups.
constexpr int kSinkSets = 16;
constexpr int kSinkLane = 256;
__device__ __attribute__((aligned(256))) char g_narrow_sink[kSinkSets * 64 * kSinkLane];

__device__ __forceinline__ void dma16(const void* g, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" : : "v"(g), "s"(lds_addr) : "memory", "m0");
}
__device__ __forceinline__ void dma4(const void* g, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dword %0, off" : : "v"(g), "s"(lds_addr) : "memory", "m0");
}
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));  // vmcnt(N)
  asm volatile("" ::: "memory");
}
__device__ __forceinline__ void wait_vm_all() { wait_vm<0>(); }
// vmcnt(6 + n) for an even n <= 40 known only at run time (else vmcnt(0))
template <int N>
__device__ __forceinline__ void wait_vm_after(int n) {
  if constexpr (N > 40) {
    wait_vm_all();
  } else {
    if (n == N) wait_vm<6 + N>();
    else wait_vm_after<N + 2>(n);
  }
}
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(reinterpret_cast<uintptr_t>(p)));
}
__device__ __forceinline__ int32_t uni(int32_t v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a, b}, bf16x2_t));
}

// The contraction of the forward tile (row type i, output group j) as at
// most two contiguous K ranges [a0, a0 + l0) and [a1, a1 + l1): B(i, j) is
// {i, j} for the star law (the graph law: {i} on the diagonal, {i, j} on an
// edge, nothing otherwise), every group for the dense law, and for the
// tensor square at most two runs of consecutive groups.
// `S(x)`: the start of input group x (x <= q).
template <typename SF>
__device__ __forceinline__ void fwd_ranges(const NarrowParams& p, SF S, int i, int j, int32_t& a0, int32_t& l0,
                                           int32_t& a1, int32_t& l1) {
  a0 = l0 = a1 = l1 = 0;
  if (p.law == 1) {
    l0 = p.K;
    return;
  }
  if (p.law == 2) {
    int lo0, hi0, lo1, hi1;
    mask_ranges(tensor_mask(kModeFwd, p.q, i, j), lo0, hi0, lo1, hi1);
    a0 = S(lo0);
    l0 = S(hi0) - a0;
    a1 = S(lo1);
    l1 = S(hi1) - a1;
    return;
  }
  if (p.law == 3 && i != j && !((p.adj[i] >> j) & 1ull)) return;  // not a slot of the row
  const int lo = min(i, j), hi = max(i, j);
  a0 = S(lo);
  l0 = S(lo + 1) - a0;
  if (hi != lo) {
    a1 = S(hi);
    l1 = S(hi + 1) - a1;
  }
}

// LDS layouts.  A: 64 rows x 64 K (128 bytes a row), 16-byte chunk c of row r
// at chunk c ^ (r & 7).  B: 64 K rows x 128 columns (256 bytes a row), chunk c
// of K row k at chunk c ^ 2 (k & 3).  Both keep the MFMA operand reads free of
// bank conflicts (a row-contiguous read of 8 rows, a transposing read of 4).
__device__ __forceinline__ int a_off(int r, int c) { return r * 128 + ((c ^ (r & 7)) << 4); }
__device__ __forceinline__ int b_off(int k, int c) { return k * 256 + ((c ^ (2 * (k & 3))) << 4); }

// A per-lane table of kMaxQFwd entries in four chunks of 64 (chunk c, lane
// l: entry 64 c + l), held in named registers: chunks are reached by
// compile-time index (get) or through scalars (entry), never by address, so
// the table never moves to scratch memory.
struct Ch4 {
  int32_t v0 = 0, v1 = 0, v2 = 0, v3 = 0;
  template <int C>
  __device__ __forceinline__ int32_t& get() {
    if constexpr (C == 0) return v0;
    else if constexpr (C == 1) return v1;
    else if constexpr (C == 2) return v2;
    else return v3;
  }
  // entry 64 c + l (uniform) of a table of NCH chunks: every chunk's lane l
  // read into a scalar, then the scalar selected (a select of the vectors
  // could be turned into an indexed access of a stack copy)
  template <int NCH>
  __device__ __forceinline__ int32_t entry(int c, int l) const {
    if constexpr (NCH == 1) {
      return __builtin_amdgcn_readlane(v0, l);
    } else {
      const int32_t e0 = __builtin_amdgcn_readlane(v0, l), e1 = __builtin_amdgcn_readlane(v1, l);
      const int32_t e2 = __builtin_amdgcn_readlane(v2, l), e3 = __builtin_amdgcn_readlane(v3, l);
      return c == 0 ? e0 : (c == 1 ? e1 : (c == 2 ? e2 : e3));
    }
  }
};
static_assert(kMaxQFwd == 4 * 64, "four chunks of 64");
// f(chunk) for the first NCH chunks (1: q <= 64, 4: q <= 256)
template <int NCH, typename F>
__device__ __forceinline__ void each_chunk(F&& f) {
  f(std::integral_constant<int, 0>{});
  if constexpr (NCH > 1) {
    f(std::integral_constant<int, 1>{});
    f(std::integral_constant<int, 2>{});
    f(std::integral_constant<int, 3>{});
  }
}

// A tile of the list: rows [pos0, pend) of the plan, columns [cstart, cend),
// the K ranges of its contraction and its K steps (0: nothing to do).
struct NTile {
  int32_t pos0, pend, cstart, cend, nsteps;
  int32_t a0, l0, a1, l1;
};

// The fp32 epilogue of one tile for one lane: row 32 wr + lr of the tile (`row`
// in the output, `rok` whether it exists), columns 64 wc + 32 cb + 8 a +
// 4 lh + 0..3 for cb < 2, a < 4.  Every lane stores all 8 blocks (and 8 of Z
// when asked for): blocks without an element go to the lane's sink.
// Y_out (with activation `act`) and Z_out (pre-activation) may be null.
__device__ __forceinline__ void narrow_epilogue(const NarrowParams& p, const f32x16_t (&acc)[2], bool rok, int32_t row,
                                                int32_t cstart, int32_t cend, int cl0, const float* bias_tile,
                                                char* sink, void* Y_out, void* Z_out, int act) {
  constexpr int esz = 4;
  const int64_t off = (static_cast<int64_t>(row) * p.N + cstart + cl0) * esz;
  char* yb = Y_out ? (rok ? static_cast<char*>(Y_out) + off : sink) : nullptr;
  char* zb = Z_out ? (rok ? static_cast<char*>(Z_out) + off : sink) : nullptr;
  const bool full = cend - cstart == kNCols;
#pragma unroll
  for (int cb = 0; cb < 2; ++cb)
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      const int cl = cl0 + 32 * cb + 8 * a;
      const int bo = (32 * cb + 8 * a) * esz;
      const bool cok = full || cstart + cl < cend;
      float v[4];
#pragma unroll
      for (int x = 0; x < 4; ++x) v[x] = acc[cb][4 * a + x];
      if (p.bias) {
        const float4 bv = *reinterpret_cast<const float4*>(bias_tile + cl);
        v[0] += bv.x; v[1] += bv.y; v[2] += bv.z; v[3] += bv.w;
      }
      auto put = [&](char* base) {
        *reinterpret_cast<float4*>((cok ? base : sink) + bo) = make_float4(v[0], v[1], v[2], v[3]);
      };
      if (zb) put(zb);
      if (act != kActNone) {
#pragma unroll
        for (int x = 0; x < 4; ++x) v[x] = act_apply(act, v[x]);
      }
      if (yb) put(yb);
    }
}

template <int NCH>
__global__ __launch_bounds__(kNThreads) void gemm_narrow_kernel(const NarrowParams p, int32_t n_ct, int32_t wg_per_xcd,
                                                                 int32_t band) {
  extern __shared__ __attribute__((aligned(16))) char smem[];  // kNStages stages of (A, B)
  __shared__ int32_t rows_s[kSlots][kNRows];                    // plan positions of the tile's rows
  __shared__ __attribute__((aligned(16))) float bias_s[kSlots][256];  // the tile's bias (first kNCols)
  __shared__ __attribute__((aligned(16))) int32_t desc_s[kSlots][8];  // the tile: see schedule()

  const int lane = threadIdx.x & 63;
  const int wave = uni(threadIdx.x >> 6);
  const int wr = wave >> 1, wc = wave & 1;
  const int lr = lane & 31, lh = lane >> 5;
  const int q = p.q;

  // Per-type and per-group tables in registers, in chunks of 64 (chunk c,
  // lane l: type or group 64 c + l), so that describing a tile reads no
  // memory: the plan offsets and the running count of 64-row blocks of the
  // types; the input group starts, output group starts and column-tile
  // prefix of the groups, and that prefix one group on (past the last
  // group: no tile reaches it).  Entry q of the starts is K, N or M.
  Ch4 off, incl, s0, r0, ntp0, ntp1;
  int32_t n_blocks = 0;
  const int32_t off_end = p.offsets[q];
  each_chunk<NCH>([&](auto C) {
    constexpr int c = decltype(C)::value;
    const int t = 64 * c + lane;
    int32_t v = 0;
    ntp1.get<c>() = 0x7fffffff;
    if (t < q) {
      off.get<c>() = p.offsets[t];
      v = (p.offsets[t + 1] - p.offsets[t] + kNRows - 1) / kNRows;
      s0.get<c>() = p.S[t];
      r0.get<c>() = p.R[t];
      ntp0.get<c>() = p.NTp[t];
      if (t + 1 < q) ntp1.get<c>() = p.NTp[t + 1];
    }
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int32_t u = __shfl_up(v, d);
      if (lane >= d) v += u;
    }
    incl.get<c>() = n_blocks + v;
    n_blocks += __builtin_amdgcn_readlane(v, 63);
  });
  // entry x of a table (x < q), else `end`
  auto pick = [&](const Ch4& tab, int x, int32_t end) -> int32_t {
    if (x >= q) return end;
    return tab.template entry<NCH>(x >> 6, x & 63);
  };

  // The tiles: (row block rb, column tile ct), the row blocks numbered type
  // by type (block rb is type i's, the first whose running block count
  // passes rb).  XCD x (workgroup w runs on XCD w mod 8) owns a region: an
  // eighth of the row blocks with every column tile, or, with fewer than 8
  // row blocks, every row block with an eighth of the column tiles.  Within
  // it the row blocks go in bands of `band` (rows whose X fits in a part of
  // the XCD's L2) and each band runs column tile by column tile, its row
  // blocks side by side: a weight tile is fetched once per band (the
  // diagonal blocks, which every type reads, once per band instead of once
  // per type) and the band's rows stay in L2.  The region's workgroups take
  // every wg_per_xcd-th item.
  const int xcd = blockIdx.x & 7;
  int32_t rb0 = 0, rb1 = n_blocks, ct0 = 0, ct1 = n_ct;
  if (n_blocks >= 8) {
    rb0 = xcd * n_blocks / 8;
    rb1 = (xcd + 1) * n_blocks / 8;
  } else {
    ct0 = xcd * n_ct / 8;
    ct1 = (xcd + 1) * n_ct / 8;
  }
  const int32_t nrb = rb1 - rb0, nct = ct1 - ct0;
  const int32_t band_items = band * nct;
  auto decode = [&](int32_t item) -> NTile {
    NTile t;
    const int32_t bi = item / band_items;
    const int32_t within = item - bi * band_items;
    const int32_t bsz = min(band, nrb - bi * band);
    const int32_t cl = within / bsz;
    const int32_t rb = rb0 + bi * band + (within - cl * bsz);
    const int32_t ct = ct0 + cl;
    int i = -1;  // the type: the first whose running block count passes rb
    each_chunk<NCH>([&](auto C) {
      constexpr int c = decltype(C)::value;
      const uint64_t m = __ballot(64 * c + lane < q && incl.get<c>() > rb);
      if (i < 0 && m) i = 64 * c + __builtin_ctzll(m);
    });
    const int32_t o_i = pick(off, i, off_end), o_i1 = pick(off, i + 1, off_end);
    const int32_t blk = rb - (pick(incl, i, 0) - (o_i1 - o_i + kNRows - 1) / kNRows);
    t.pos0 = o_i + blk * kNRows;
    t.pend = min(o_i1, t.pos0 + kNRows);
    int j = 0;  // the output group: column tiles at or past the next groups' prefixes
    each_chunk<NCH>([&](auto C) { j += __popcll(__ballot(ct >= ntp1.get<decltype(C)::value>())); });
    t.cstart = pick(r0, j, p.N) + (ct - pick(ntp0, j, n_ct)) * kNCols;
    t.cend = min(pick(r0, j + 1, p.N), t.cstart + kNCols);
    fwd_ranges(p, [&](int x) { return pick(s0, x, p.K); }, i, j, t.a0, t.l0, t.a1, t.l1);
    t.nsteps = (t.l0 + t.l1 + kNK - 1) / kNK;
    return t;
  };
  const int32_t last = nrb * nct;
  int32_t s_item = blockIdx.x >> 3;

  const uint16_t* X = static_cast<const uint16_t*>(p.A);
  const uint16_t* W = static_cast<const uint16_t*>(p.B);
  const void* zero = g_narrow_zero;
  const uint32_t smem_base = lds_addr(smem);

  // ---- scheduler (wave 0): the n-th tile of this workgroup is described in
  // slot n mod kSlots, kSlots - 1 tiles ahead of the consumer: its row count,
  // columns, steps and group mask, with the plan positions of its rows and
  // its bias copied straight into LDS (lanes past the rows or columns, and
  // every lane without a bias, copy zeros: always 2 copies).  A tile of no
  // steps ends the list.  The producer reaches a tile at least two
  // iterations after it was described, so the copies issued for it are
  // older than the element copies waited for by then.
  int32_t s_n = 0;
  auto schedule = [&]() {
    if (wave != 0) return;
    NTile t;
    t.nsteps = 0;
    for (; s_item < last; s_item += wg_per_xcd) {
      t = decode(s_item);
      if (t.nsteps > 0) break;
    }
    const int slot = s_n % kSlots;
    if (s_item < last) {
      s_item += wg_per_xcd;
    } else {
      t.nsteps = 0;
      t.pos0 = t.pend = t.cstart = t.cend = 0;
      t.a0 = t.l0 = t.a1 = t.l1 = 0;
    }
    dma4(lane < t.pend - t.pos0 ? static_cast<const void*>(p.perm + t.pos0 + lane) : zero, lds_addr(rows_s[slot]));
    dma16(p.bias && t.cstart + 4 * lane < t.cend ? static_cast<const void*>(p.bias + t.cstart + 4 * lane) : zero,
          lds_addr(bias_s[slot]));
    if (lane == 0) {
      *reinterpret_cast<int4*>(desc_s[slot]) = make_int4(t.pend - t.pos0, t.cstart, t.cend, t.nsteps);
      *reinterpret_cast<int4*>(desc_s[slot] + 4) = make_int4(t.a0, t.l0, t.a1, t.l1);
    }
    ++s_n;
  };

  // ---- producer: the stream of (tile, K step) elements, copied
  // kNStages - 1 elements ahead of the consumer; every element is 6 copies
  // per wave (2 of A, 4 of B).  A tile's descriptor is read when its first
  // element is copied (a barrier after the scheduler wrote it); the copy
  // sources of its A rows and B columns are set up then.  Step s covers
  // positions [64 s, 64 s + 64) of the concatenated K ranges: a lane's
  // position below l0 reads K = a0 + position, below l0 + l1 K = a1 +
  // position - l0, past that zeros (8-wide A chunks never span the two
  // ranges: the widths are multiples of 8).  Rows past the tile's read row 0
  // and columns past it read the group's last columns: their products are
  // never stored.
  int32_t p_n = 0, p_s = 0, p_nsteps = 0, p_a0 = 0, p_l0 = 0, p_a1 = 0, p_len = 0;
  bool p_fresh = true, p_done = false;
  const uint16_t* abase[2];
  const uint16_t* bbase[4];
  auto produce = [&](int stage) -> bool {
    if (p_fresh) {
      p_fresh = false;
      const int4 d0 = *reinterpret_cast<const int4*>(desc_s[p_n % kSlots]);
      const int4 d1 = *reinterpret_cast<const int4*>(desc_s[p_n % kSlots] + 4);
      p_nsteps = uni(d0.w);
      if (p_nsteps == 0) {
        p_done = true;
      } else {
        const int32_t cstart = uni(d0.y);
        p_a0 = uni(d1.x);
        p_l0 = uni(d1.y);
        p_a1 = uni(d1.z);
        p_len = p_l0 + uni(d1.w);
        p_s = 0;
        const int32_t* rows = rows_s[p_n % kSlots];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const int r = 8 * (wave + 4 * u) + (lane >> 3), c = (lane & 7) ^ (r & 7);
          abase[u] = X + static_cast<int64_t>(rows[r]) * p.K + 8 * c;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int kr = 4 * (wave + 4 * u) + (lane >> 4), c = (lane & 15) ^ (2 * (kr & 3));
          const int32_t col = min(cstart + 8 * c, p.N - 8);
          bbase[u] = W + static_cast<int64_t>(kr) * p.N + col;
        }
      }
    }
    if (p_done) return false;
    const uint32_t As = smem_base + stage * kStage, Bs = As + kA;
    const int32_t pos = kNK * p_s;
    const int32_t k0 = p_a0 + pos, k1 = p_a1 - p_l0 + pos;  // K of position pos + x: k0 + x or k1 + x
    if (pos + kNK <= p_l0 || (pos >= p_l0 && pos + kNK <= p_len)) {  // the step lies in one range
      const int32_t k = pos + kNK <= p_l0 ? k0 : k1;
      const int64_t kofs = static_cast<int64_t>(k) * p.N;
#pragma unroll
      for (int u = 0; u < 2; ++u) dma16(abase[u] + k, As + (wave + 4 * u) * 1024);
#pragma unroll
      for (int u = 0; u < 4; ++u) dma16(bbase[u] + kofs, Bs + (wave + 4 * u) * 1024);
    } else {  // the step spans both ranges or runs past the end
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int r = 8 * (wave + 4 * u) + (lane >> 3), x = 8 * ((lane & 7) ^ (r & 7));
        const int32_t k = pos + x < p_l0 ? k0 : k1;
        dma16(pos + x < p_len ? static_cast<const void*>(abase[u] + k) : zero, As + (wave + 4 * u) * 1024);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int x = 4 * (wave + 4 * u) + (lane >> 4);
        const int32_t k = pos + x < p_l0 ? k0 : k1;
        dma16(pos + x < p_len ? static_cast<const void*>(bbase[u] + static_cast<int64_t>(k) * p.N) : zero,
              Bs + (wave + 4 * u) * 1024);
      }
    }
    if (++p_s == p_nsteps) {
      ++p_n;
      p_fresh = true;
    }
    return true;
  };

  // ---- prologue: the first kSlots - 1 tiles described, then the first
  // kNStages - 1 elements copied
  for (int n = 0; n < kSlots - 1; ++n) schedule();
  wait_vm_all();
  __syncthreads();
  bool ahead = false;  // whether the element after the consumer's was copied
  for (int e = 0; e < kNStages - 1; ++e) ahead = produce(e);

  // ---- consumer
  auto read_tile = [&](int n, int32_t& nrows, int32_t& cstart, int32_t& cend, int32_t& nsteps) {
    const int4 d0 = *reinterpret_cast<const int4*>(desc_s[n % kSlots]);
    nrows = uni(d0.x);
    cstart = uni(d0.y);
    cend = uni(d0.z);
    nsteps = uni(d0.w);
  };
  int32_t c_n = 0, c_s = 0, c_nrows, c_cstart, c_cend, c_nsteps;
  read_tile(0, c_nrows, c_cstart, c_cend, c_nsteps);
  f32x16_t acc[2];
  const int g = lane >> 4, pp = lane & 15;
  const int rr = pp >> 2, qq = pp & 3;
  char* sink = g_narrow_sink + ((blockIdx.x % kSinkSets) * 64 + lane) * kSinkLane;
  // stores of the output blocks at the ends of the last two iterations and
  // the scheduler's copies of the last one (issued after the copies of this
  // iteration's element); per tile each lane stores 4 chunks of 16 bytes of
  // a bf16 output, 8 blocks of an fp32 one, and as many again of Z
  // (SwiGLU: half as many of H, plus those of Z when asked for)
  const int n_st = p.swiglu ? (p.ydtype == 0 ? 4 + (p.Z ? 8 : 0) : 2 + (p.Z ? 4 : 0))
                            : (p.ydtype == 0 ? 8 : 4) * (p.Z ? 2 : 1);
  int st1 = 0, st2 = 0, sd1 = 0;
  for (int32_t e = 0; c_nsteps > 0; ++e) {
    // Memory operations complete in order for the counter: element e's
    // copies have landed once no more are outstanding than were issued after
    // them: the 6 copies of element e + 1, the stores of the last two
    // iterations and the scheduler's copies of the last one.
    const int after = st1 + st2 + sd1;
    if (!ahead) wait_vm_all();
    else wait_vm_after<0>(after);
    st2 = st1;
    st1 = 0;
    sd1 = 0;
    __syncthreads();  // element e and the scheduler's last writes are visible;
                      // element e - 1 and the tile before this one are done with
    const bool first = c_s == 0;
    if (first) {
      schedule();  // tile c_n + 4, into the slot of tile c_n - 1
      if (wave == 0) sd1 = 2;
    }
    ahead = produce((e + kNStages - 1) % kNStages);
    const char* As = smem + (e % kNStages) * kStage;
    const char* Bs = As + kA;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      // B operand of the C^T block: 8 consecutive K of row 32 wr + lr
      const uint4 xf = *reinterpret_cast<const uint4*>(As + a_off(32 * wr + lr, 2 * ks + lh));
#pragma unroll
      for (int cb = 0; cb < 2; ++cb) {
        // A operand: 8 consecutive K of column 64 wc + 32 cb + lr, by two
        // transposing reads of 4 K rows each
        const int col = 64 * wc + 32 * cb + 16 * (g & 1) + 4 * qq;  // this lane's 4 addressed columns
        const int k1 = 16 * ks + 8 * (g >> 1) + rr;
        const char* a0 = Bs + b_off(k1, col >> 3) + ((col >> 2) & 1) * 8;
        const char* a1 = Bs + b_off(k1 + 4, col >> 3) + ((col >> 2) & 1) * 8;
        const uint2 w0 = __builtin_bit_cast(uint2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((STARQ_LDS v4i16_t*)(a0)));
        const uint2 w1 = __builtin_bit_cast(uint2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((STARQ_LDS v4i16_t*)(a1)));
        const bf16x8_t wf = __builtin_bit_cast(bf16x8_t, make_uint4(w0.x, w0.y, w1.x, w1.y));
        if (ks == 0 && first)
          acc[cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf, __builtin_bit_cast(bf16x8_t, xf), f32x16_t{}, 0, 0, 0);
        else
          acc[cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf, __builtin_bit_cast(bf16x8_t, xf), acc[cb], 0, 0, 0);
      }
    }
    if (++c_s < c_nsteps) continue;
    // ---- epilogue of the tile
    {
      const int r = 32 * wr + lr;
      const bool rok = r < c_nrows;
      const int32_t row = rows_s[c_n % kSlots][r];
      const float* bt = bias_s[c_n % kSlots];
      if (p.ydtype == 0) {
        if (!p.swiglu) narrow_epilogue(p, acc, rok, row, c_cstart, c_cend, 64 * wc + 4 * lh, bt, sink, p.Y, p.Z, p.act);
        else if (p.Z) narrow_epilogue(p, acc, rok, row, c_cstart, c_cend, 64 * wc + 4 * lh, bt, sink, nullptr, p.Z, 0);
      } else {
        // bf16 through LDS, in the stage this iteration consumed (free until
        // the next iteration's copies): the 64 x 128 values go in with row r
        // at r * 256 bytes and 16-byte chunk c at c ^ (r & 15), then each
        // thread stores 16-byte chunks of whole rows (16 lanes a row)
        char* T = smem + (e % kNStages) * kStage;
        const int32_t* rows = rows_s[c_n % kSlots];
        auto pass = [&](void* out, bool activate) {
          __syncthreads();  // every wave is done reading the stage (or the last pass)
#pragma unroll
          for (int cb = 0; cb < 2; ++cb)
#pragma unroll
            for (int a = 0; a < 4; ++a) {
              const int cl = 64 * wc + 32 * cb + 8 * a + 4 * lh;
              float v[4];
#pragma unroll
              for (int x = 0; x < 4; ++x) v[x] = acc[cb][4 * a + x];
              if (p.bias) {
                const float4 bv = *reinterpret_cast<const float4*>(bt + cl);
                v[0] += bv.x; v[1] += bv.y; v[2] += bv.z; v[3] += bv.w;
              }
              if (activate) {
#pragma unroll
                for (int x = 0; x < 4; ++x) v[x] = act_apply(p.act, v[x]);
              }
              *reinterpret_cast<uint2*>(T + r * 256 + (((cl >> 3) ^ (r & 15)) << 4) + ((cl >> 2) & 1) * 8) =
                  make_uint2(pack_bf16(v[0], v[1]), pack_bf16(v[2], v[3]));
            }
          __syncthreads();
#pragma unroll
          for (int it = 0; it < 4; ++it) {
            const int id = threadIdx.x + kNThreads * it, tr = id >> 4, c = id & 15;
            const uint4 val = *reinterpret_cast<const uint4*>(T + tr * 256 + ((c ^ (tr & 15)) << 4));
            const bool ok = tr < c_nrows && c_cstart + 8 * c < c_cend;
            const int64_t off = (static_cast<int64_t>(rows[tr]) * p.N + c_cstart + 8 * c) * 2;
            *reinterpret_cast<uint4*>(ok ? static_cast<char*>(out) + off : sink + 16 * it) = val;
          }
        };
        if (p.Z) pass(p.Z, false);
        if (!p.swiglu) pass(p.Y, p.act != kActNone);
      }
      if (p.swiglu) {
        // H = silu(gate) . up: columns alternate 8 gate, 8 up, so the
        // lane's block a = 2 pp holds gate values and a = 2 pp + 1 the up
        // values of the same features: H feature
        // 32 wc + 16 cb + 8 pp + 4 lh + x of the tile, column c_cstart / 2 +
        // that of H [M, N / 2]
        float h[4][4];  // [2 cb + pp][x]
#pragma unroll
        for (int cb = 0; cb < 2; ++cb)
#pragma unroll
          for (int pp2 = 0; pp2 < 2; ++pp2)
#pragma unroll
            for (int x = 0; x < 4; ++x) {
              const int cl = 64 * wc + 32 * cb + 16 * pp2 + 4 * lh + x;
              float g = acc[cb][8 * pp2 + x], u = acc[cb][8 * pp2 + 4 + x];
              if (p.bias) {
                g += bt[cl];
                u += bt[cl + 8];
              }
              h[2 * cb + pp2][x] = g * sigmoid_fast(g) * u;
            }
        const int32_t hn = p.N / 2, hw = (c_cend - c_cstart) / 2;  // H row width, the tile's H columns
        if (p.ydtype == 0) {  // fp32: from the registers
          const int64_t off = (static_cast<int64_t>(row) * hn + c_cstart / 2 + 32 * wc + 4 * lh) * 4;
#pragma unroll
          for (int b = 0; b < 4; ++b) {  // feature 32 wc + 8 b + 4 lh + 0..3
            const bool ok = rok && 32 * wc + 8 * b + 4 * lh < hw;
            *reinterpret_cast<float4*>((ok ? static_cast<char*>(p.Y) + off : sink) + 32 * b) =
                make_float4(h[b][0], h[b][1], h[b][2], h[b][3]);
          }
        } else {  // bf16: 64 rows x 64 features through LDS, 16-byte chunks of whole rows
          char* T = smem + (e % kNStages) * kStage;
          const int32_t* rows = rows_s[c_n % kSlots];
          __syncthreads();  // every wave is done reading the stage (or the Z pass)
#pragma unroll
          for (int b = 0; b < 4; ++b) {
            const int fl = 32 * wc + 8 * b + 4 * lh;
            *reinterpret_cast<uint2*>(T + r * 128 + (((fl >> 3) ^ (r & 7)) << 4) + ((fl >> 2) & 1) * 8) =
                make_uint2(pack_bf16(h[b][0], h[b][1]), pack_bf16(h[b][2], h[b][3]));
          }
          __syncthreads();
#pragma unroll
          for (int it = 0; it < 2; ++it) {
            const int id = threadIdx.x + kNThreads * it, tr = id >> 3, c = id & 7;
            const uint4 val = *reinterpret_cast<const uint4*>(T + tr * 128 + ((c ^ (tr & 7)) << 4));
            const bool ok = tr < c_nrows && 8 * c < hw;
            const int64_t off = (static_cast<int64_t>(rows[tr]) * hn + c_cstart / 2 + 8 * c) * 2;
            *reinterpret_cast<uint4*>(ok ? static_cast<char*>(p.Y) + off : sink + 16 * it) = val;
          }
        }
      }
      st1 = n_st;
    }
    ++c_n;
    c_s = 0;
    read_tile(c_n, c_nrows, c_cstart, c_cend, c_nsteps);  // written at the start of tile c_n - 4
  }
}

}  // namespace

int32_t gemm_narrow_row_blocks_upper(int64_t M, int q) { return static_cast<int32_t>(M / kNRows + q); }
int gemm_narrow_cols() { return kNCols; }

hipError_t launch_gemm_narrow(const NarrowParams& p, int32_t n_rb, int32_t n_ct, int cus, hipStream_t stream) {
  // n_rb bounds the row blocks from above (the kernel counts them from the
  // plan's offsets)
  const int64_t items = static_cast<int64_t>(n_rb) * n_ct;
  if (items <= 0 || items > 0x7fffff00 || p.N < 8) return hipErrorInvalidValue;
  // persistent: two workgroups per CU (72 KB of LDS each), the same number
  // on every XCD, no more than there are items per XCD
  const int64_t per_xcd = (items + 7) / 8;
  const int wg_per_xcd = static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(per_xcd, 2 * std::max(cus, 8) / 8)));
  static std::atomic<unsigned long long> set1{0}, set4{0};
  auto kern = p.q <= 64 ? gemm_narrow_kernel<1> : gemm_narrow_kernel<4>;
  hipError_t e = ensure_lds_limit(reinterpret_cast<const void*>(kern), p.q <= 64 ? set1 : set4, kNSmem);
  if (e != hipSuccess) return e;
  // bands of row blocks whose X rows take at most 2 MB (half an XCD's L2)
  const int32_t band = static_cast<int32_t>(std::max<int64_t>(1, (int64_t{2} << 20) / (int64_t{kNRows} * p.K * 2)));
  hipLaunchKernelGGL(kern, dim3(8 * wg_per_xcd), dim3(kNThreads), kNSmem, stream, p, n_ct, wg_per_xcd, band);
  return hipGetLastError();
}

}  // namespace starq
