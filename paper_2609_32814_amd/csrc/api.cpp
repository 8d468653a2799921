// C ABI of libstarq: argument validation, workspace layout, tile planning
// and kernel launches.  Every argument error is detected here, before any
// launch.  The only process-wide state is a read-only cache of each device's
// compute-unit count.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <initializer_list>
#include <vector>

#include "../../include/star_proj.h"
#include "kernels.hpp"

namespace {

using namespace starq;

static_assert(STAR_MAX_Q == kMaxQGroups, "one q limit for the ABI and the kernels");
static_assert(STAR_DECODE_SCRATCH_BYTES == kDecodeScratchBytes, "one size for the static decode workspace");

constexpr size_t kAlign = 256;
constexpr int64_t kMaxDim = (int64_t{1} << 30);

size_t align_up(size_t v) { return (v + kAlign - 1) & ~(kAlign - 1); }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

struct Alg {
  int q = 0;
  int law = 0;
  int64_t S[kMaxQFwd + 1];  // input group starts
  int64_t R[kMaxQFwd + 1];  // output group starts
  uint64_t adj[kMaxQGroups] = {};     // law 3: bit j of adj[i] for the edge i -> j
  uint64_t adj_in[kMaxQGroups] = {};  // law 3: bit i of adj_in[j] for the edge i -> j
  int64_t K() const { return S[q]; }
  int64_t N() const { return R[q]; }
  int64_t s(int g) const { return S[g + 1] - S[g]; }
  int64_t r(int g) const { return R[g + 1] - R[g]; }
};

// k in B(i, j) for the law (host side of the kernels' rule)
bool host_in_support(const Alg& a, int i, int j, int k) {
  if (a.law == STAR_LAW_TENSOR2) return ((k ^ i) & (k ^ j)) == 0;
  if (a.law == STAR_LAW_GRAPH) {
    if (j == i) return k == i;
    return ((a.adj[i] >> j) & 1ull) && (k == i || k == j);
  }
  return a.law == STAR_LAW_DENSE || k == i || k == j;
}

// `large`: the caller takes q up to STAR_MAX_Q_FWD (the forward product of
// the star and dense laws); elsewhere q is at most STAR_MAX_Q.
star_status parse_alg(const star_algebra* a, Alg& out, bool large = false) {
  if (!a || !a->s || !a->r) return STAR_ERR_ARG;
  if (a->q < 1 || a->q > kMaxQFwd) return STAR_ERR_ARG;
  if (a->law != STAR_LAW_STAR && a->law != STAR_LAW_DENSE && a->law != STAR_LAW_TENSOR2 &&
      a->law != STAR_LAW_GRAPH)
    return STAR_ERR_ARG;
  if (a->q > kMaxQGroups && (!large || (a->law != STAR_LAW_STAR && a->law != STAR_LAW_DENSE)))
    return STAR_ERR_UNSUPPORTED;
  if (a->law == STAR_LAW_GRAPH && !a->edges) return STAR_ERR_ARG;
  // the tensor power needs q = 2^L; the kernels take every contraction as
  // at most two contiguous group ranges, which holds for L <= 2
  if (a->law == STAR_LAW_TENSOR2 && a->q != 1 && a->q != 2 && a->q != 4) return STAR_ERR_UNSUPPORTED;
  out.q = a->q;
  out.law = a->law;
  out.S[0] = out.R[0] = 0;
  for (int g = 0; g < a->q; ++g) {
    if (a->s[g] <= 0 || a->r[g] <= 0) return STAR_ERR_SHAPE;
    if (a->s[g] % 8 || a->r[g] % 8) return STAR_ERR_ALIGN;
    out.S[g + 1] = out.S[g] + a->s[g];
    out.R[g + 1] = out.R[g] + a->r[g];
    if (out.S[g + 1] > kMaxDim || out.R[g + 1] > kMaxDim) return STAR_ERR_SHAPE;
  }
  for (int g = 0; g < kMaxQGroups; ++g) out.adj[g] = out.adj_in[g] = 0;
  if (a->law == STAR_LAW_GRAPH)
    for (int i = 0; i < a->q; ++i)
      for (int j = 0; j < a->q; ++j)
        if (i != j && a->edges[i * a->q + j]) {  // the diagonal is ignored
          out.adj[i] |= 1ull << j;
          out.adj_in[j] |= 1ull << i;
        }
  return STAR_OK;
}

bool valid_dtype(star_dtype d) { return d == STAR_F32 || d == STAR_BF16; }
bool valid_act(star_act a) {
  return a == STAR_ACT_NONE || a == STAR_ACT_GELU || a == STAR_ACT_GELU_TANH;
}

int cu_count() {
  static std::atomic<int> cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 256;
  if (dev < 64) {
    int v = cache[dev].load(std::memory_order_relaxed);
    if (v > 0) return v;
  }
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
    n = 256;
  if (dev < 64) cache[dev].store(n, std::memory_order_relaxed);
  return n;
}

// ---- workspace layouts -----------------------------------------------------

struct PlanWs {
  size_t perm = 0, offsets = 0, end = 0;
};
PlanWs plan_layout(int64_t M, int q, size_t base = 0) {
  PlanWs w;
  w.perm = base;
  w.offsets = align_up(w.perm + sizeof(int32_t) * static_cast<size_t>(std::max<int64_t>(M, 1)));
  w.end = align_up(w.offsets + sizeof(int32_t) * (q + 1));
  return w;
}

int tiles_of(int64_t w, int tile) { return static_cast<int>((w + tile - 1) / tile); }

// Column-tile width of the weight-gradient GEMM: 128 columns (the
// contraction is over rows, the output K x N is small).
constexpr int kBwdWeightNW = 2;

int bwd_weight_nsplit(const Alg& a, int64_t M) {
  int64_t mt = 0, nt = 0;
  for (int g = 0; g < a.q; ++g) {
    mt += tiles_of(a.s(g), kTileM);
    nt += tiles_of(a.r(g), 64 * kBwdWeightNW);
  }
  const int64_t base = mt * nt;
  // about one tile per CU of a 256-CU device, rows per split >= 1024
  int64_t ns = (256 + base - 1) / base;
  ns = std::min<int64_t>(ns, 8);
  ns = std::min<int64_t>(ns, std::max<int64_t>(1, M / 1024));
  return static_cast<int>(std::max<int64_t>(ns, 1));
}

// Weight gradient with bf16 operands (pipelined kernel, 256-row tiles of
// tn columns): the same rule on its own tile count.
int64_t nsplit_rule(int64_t base, int64_t M) {
  int64_t ns = (256 + base - 1) / base;
  ns = std::min<int64_t>(ns, 8);
  ns = std::min<int64_t>(ns, std::max<int64_t>(1, M / 1024));
  return std::max<int64_t>(ns, 1);
}

// Column tiles of width tn over the output groups (r) or the input groups.
int64_t col_tiles(const Alg& a, bool over_r, int tn) {
  int64_t n = 0;
  for (int g = 0; g < a.q; ++g) n += tiles_of(over_r ? a.r(g) : a.s(g), tn);
  return n;
}

// Column-tile width of the pipelined bf16 kernel: 256, or 192 (star and
// dense laws) where the launch's estimated makespan is shorter, a 192-wide
// K step counted as 0.9 of a 256-wide one (its copies and per-step costs do
// not shrink with its MFMAs).  The estimate deals the two passes' tiles (K
// steps each, in the kernel's order, rows taken as spread evenly over the
// types, as the host does not read the per-type counts) the way the kernel
// does on 256 CUs: an eighth of each pass per XCD, in snake order over the
// XCD's 32 workgroups, each tile also paying its epilogue.  Checked against
// measured pairs: 8192 x 768 -> 3072 at q = 2 (192: 512 tiles, one long and
// one short per CU), the 384-wide groups of 16384 x 3072 -> 768 (192: no
// padding), and the weight gradient 768 x 3072 over 16384 rows (256: at 192
// the split count drops to 4 and the diagonal tiles run long).
double deal_makespan(const std::vector<int32_t>* passes, double epi) {
  constexpr int kGrid = 256, kSlots = kGrid / 8;
  double worst = 0.0;
  for (int x = 0; x < 8; ++x) {
    double load[kSlots] = {};
    int64_t v = 0;
    for (int ps = 0; ps < 2; ++ps) {
      const int64_t n = static_cast<int64_t>(passes[ps].size()), chunk = (n + 7) / 8;
      for (int64_t t = x * chunk; t < std::min(n, (x + 1) * chunk); ++t, ++v) {
        const int64_t r = v / kSlots, pos = v % kSlots;
        load[(r & 1) ? kSlots - 1 - pos : pos] += passes[ps][t] + epi;
      }
    }
    for (double l : load) worst = std::max(worst, l);
  }
  return worst;
}
int steps_of(int64_t w) { return static_cast<int>((w + 63) / 64); }
// mode: the kernel's (forward, activation gradient, weight gradient); tm
// the tile height (the weight gradient's, over the input groups)
double async_makespan(const Alg& a, int mode, int64_t M, int tm, int tn, bool act) {
  std::vector<int32_t> passes[2];
  const int q = a.q;
  const int64_t per = (M + q - 1) / q;  // rows of a type
  if (mode == kModeBwdWeight) {
    int64_t mt = 0;
    for (int g = 0; g < q; ++g) mt += tiles_of(a.s(g), tm);
    const int64_t ns = nsplit_rule(mt * col_tiles(a, true, tn), M);
    for (int i = 0; i < q; ++i)
      for (int j = 0; j < q; ++j) {
        const bool diag = i == j || a.law == STAR_LAW_DENSE;
        const int st = steps_of(((diag ? M : per) + ns - 1) / ns);
        passes[i == j ? 0 : 1].insert(passes[i == j ? 0 : 1].end(), tiles_of(a.s(i), tm) * tiles_of(a.r(j), tn) * ns,
                                      st);
      }
    return deal_makespan(passes, 1.0 * tm * tn / (256 * 256));
  }
  const int rt = tiles_of(per, kTileM);
  const bool fwd = mode == kModeFwd;
  for (int i = 0; i < q; ++i)
    for (int u = 0; u < rt; ++u)
      for (int j = 0; j < q; ++j) {
        const int ct = tiles_of(fwd ? a.r(j) : a.s(j), tn);
        int st;
        if (a.law == STAR_LAW_DENSE) st = steps_of(fwd ? a.K() : a.N());
        else if (fwd) st = steps_of(a.s(j)) + (j != i ? steps_of(a.s(i)) : 0);
        else st = j == i ? steps_of(a.N()) : steps_of(a.r(j));
        // pass 0: forward, the two-segment tiles; activation gradient, the
        // tiles over every output group
        const int ps = a.law == STAR_LAW_DENSE ? 0 : (fwd ? (j != i ? 0 : 1) : (j == i ? 0 : 1));
        passes[ps].insert(passes[ps].end(), ct, st);
      }
  const double epi = (act ? (fwd ? 3.0 : 2.0) : 1.0) * tn / 256;
  return deal_makespan(passes, epi);
}
// The default takes 192 only where it pads fewer C columns as well: without
// padding to remove, the 192-wide tiles' extra re-reads of the row tiles
// (a third more column tiles per row tile) made them slower on row types in
// short runs (192 rows: 78 against 63 us for the dense 8192 x 768 -> 3072),
// even where the deal favours them (1024-row runs: 57 against 63 us).
int padded_cols(const Alg& a, bool over_r, int tn) {
  return static_cast<int>(col_tiles(a, over_r, tn) * tn);
}
int async_tile_n(const Alg& a, int mode, int64_t M, bool act) {
  if (a.law != STAR_LAW_STAR && a.law != STAR_LAW_DENSE) return 256;
  const bool over_r = mode != kModeBwdData;
  if (padded_cols(a, over_r, 192) >= padded_cols(a, over_r, 256)) return 256;
  return 0.9 * async_makespan(a, mode, M, 256, 192, act) < async_makespan(a, mode, M, 256, 256, act) ? 192 : 256;
}
// Weight gradient: 256 x 256, 256 x 192 (columns over 384-wide output
// groups) or 192 x 256 (rows over 384-wide input groups), the one that pads
// the fewest dW cells, if the deal estimate agrees (a smaller tile counted
// as 0.9 of a 256 x 256 one per step).
struct TileShape {
  int tm, tn;
};
TileShape async_tiles_weight(const Alg& a, int64_t M) {
  if (a.law != STAR_LAW_STAR && a.law != STAR_LAW_DENSE) return {256, 256};
  auto padded = [&](int tm, int tn) {
    int64_t rows = 0;
    for (int g = 0; g < a.q; ++g) rows += static_cast<int64_t>(tiles_of(a.s(g), tm)) * tm;
    return rows * padded_cols(a, true, tn);
  };
  const double base = async_makespan(a, kModeBwdWeight, M, 256, 256, false);
  TileShape best{256, 256};
  int64_t best_pad = padded(256, 256);
  for (const TileShape c : {TileShape{256, 192}, TileShape{192, 256}}) {
    const int64_t pad = padded(c.tm, c.tn);
    if (pad < best_pad && 0.9 * async_makespan(a, kModeBwdWeight, M, c.tm, c.tn, false) < base) {
      best = c;
      best_pad = pad;
    }
  }
  return best;
}
int bwd_weight_nsplit_async(const Alg& a, int64_t M) {
  const TileShape ts = async_tiles_weight(a, M);
  int64_t mt = 0;
  for (int g = 0; g < a.q; ++g) mt += tiles_of(a.s(g), ts.tm);
  return static_cast<int>(nsplit_rule(mt * col_tiles(a, true, ts.tn), M));
}

constexpr int kColSumChunks = 64;  // row chunks of the bias-gradient column sums

// Workspace of the weight gradient: the plan, then either the fp32 path's
// split partials or the bf16 path's split partials and bias-gradient chunk
// sums (the two paths share the space).
struct BwdWs {
  PlanWs plan;
  int nsplit = 1;
  size_t partial = 0, dbias_part = 0;
  int nsplit_a = 1;
  size_t partial_a = 0, colsum = 0;
  size_t end = 0;
};
BwdWs bwd_weight_layout(const Alg& a, int64_t M) {
  BwdWs w;
  w.plan = plan_layout(M, a.q);
  w.nsplit = bwd_weight_nsplit(a, M);
  size_t cur = w.plan.end;
  if (w.nsplit > 1) {
    w.partial = cur;
    cur = align_up(cur + sizeof(float) * static_cast<size_t>(w.nsplit) * a.K() * a.N());
    w.dbias_part = cur;
    cur = align_up(cur + sizeof(float) * static_cast<size_t>(w.nsplit) * a.N());
  }
  const size_t end32 = cur;
  w.nsplit_a = bwd_weight_nsplit_async(a, M);
  cur = w.plan.end;
  if (w.nsplit_a > 1) {
    w.partial_a = cur;
    cur = align_up(cur + sizeof(float) * static_cast<size_t>(w.nsplit_a) * a.K() * a.N());
  }
  w.colsum = cur;
  cur = align_up(cur + sizeof(float) * static_cast<size_t>(kColSumChunks) * a.N());
  w.end = std::max(end32, cur);
  return w;
}

// Every decode workspace starts with the status line: the decode stack's
// error flag (int32 at offset 0, raised when one of its bounded waits ran
// out) on a 256-byte line of its own, zeroed by every star_decode call and
// read by star_decode_status.
constexpr size_t kDecodeStatusBytes = kCounterStride * sizeof(int32_t);

struct DecodeWs {
  size_t h = 0, xb = 0, H = 0, end = 0;
};
DecodeWs decode_layout(const Alg& up, int64_t M) {
  DecodeWs w;
  const int64_t D = up.K(), F = up.N();
  size_t cur = kDecodeStatusBytes;
  w.h = cur;
  cur = align_up(cur + sizeof(float) * M * D);
  w.xb = cur;
  cur = align_up(cur + sizeof(uint16_t) * M * D);
  w.H = cur;
  cur = align_up(cur + sizeof(uint16_t) * M * F);
  w.end = cur;
  return w;
}

// The single-launch decode stack: 16-column tiles of F (up) and of D (down),
// the down contraction over F cut into ns chunks so both phases have about
// as many items; usable when every item's inputs and two weight slots fit
// in LDS, the grid fits on the device at one workgroup per CU and the layer
// pointers fit in the kernel arguments.  Layout: the counters (the first of
// them the status line) and the tagged hand-off words first, so that one
// fill clears them all, then H, the bf16 inputs, h and the down partials.
struct StackPlan {
  bool ok = false;
  int ns = 1, kc = 0, nt_up = 0, nt_dn = 0, grid = 0;
  size_t H = 0, hb = 0, h = 0, part = 0, tH = 0, tpart = 0, cnt = 0, zero_end = 0, end = 0;
  bool resident = false;
};
StackPlan stack_plan(const Alg& u, const Alg& d, int64_t M, int n_layers, bool gated = false) {
  StackPlan sp;
  const int64_t D = u.K(), F = u.N();
  for (int g = 0; g < u.q; ++g) sp.nt_up += static_cast<int>(tiles_of(u.r(g), kDecodeTileN));
  for (int g = 0; g < d.q; ++g) sp.nt_dn += static_cast<int>(tiles_of(d.r(g), kDecodeTileN));
  sp.ns = static_cast<int>(std::max<int64_t>(1, (sp.nt_up + sp.nt_dn - 1) / sp.nt_dn));
  sp.kc = static_cast<int>((F + sp.ns - 1) / sp.ns);
  sp.kc = (sp.kc + 127) / 128 * 128;
  sp.ns = static_cast<int>((F + sp.kc - 1) / sp.kc);
  sp.grid = std::max(sp.nt_up, sp.nt_dn * sp.ns);
  const int kmax = static_cast<int>(std::max<int64_t>(D, sp.kc));
  sp.resident = M >= 1 && M <= kDecodeMaxRows &&
                decode_stack_resident(static_cast<int>(M), kmax, static_cast<int>(D), sp.ns, gated, sp.nt_up,
                                      sp.nt_dn);
  size_t cur = 0;
  sp.cnt = cur;
  cur = align_up(cur + sizeof(int32_t) * decode_stack_counters(sp.nt_dn));
  sp.tH = cur;
  sp.tpart = cur;
  if (sp.resident) {
    cur = align_up(cur + sizeof(uint64_t) * M * (F / 2));
    sp.tpart = cur;
    cur = align_up(cur + sizeof(uint64_t) * 2 * sp.ns * M * D);
  }
  sp.zero_end = cur;
  sp.H = cur;
  cur = align_up(cur + sizeof(uint16_t) * M * F);
  sp.hb = cur;
  cur = align_up(cur + 2 * sizeof(uint16_t) * M * D);
  sp.h = cur;
  cur = align_up(cur + sizeof(float) * M * D);
  sp.part = cur;
  cur = align_up(cur + sizeof(float) * sp.ns * M * D);
  sp.end = cur;
  bool same_groups = u.q == d.q && u.law == d.law;
  for (int g = 0; same_groups && g <= u.q; ++g) same_groups = d.S[g] == u.R[g] && d.R[g] == u.S[g];
  // one support table for both projections (the graph law: the same graph)
  for (int g = 0; same_groups && g < u.q; ++g) same_groups = u.adj[g] == d.adj[g];
  sp.ok = M >= 1 && M <= kDecodeMaxRows && n_layers <= kStackMaxLayers && same_groups &&
          decode_stack_smem(static_cast<int>(M), kmax, static_cast<int>(D), sp.ns, gated) > 0 &&
          sp.grid <= cu_count();
  return sp;
}

template <typename T>
T* at(void* ws, size_t off) {
  return reinterpret_cast<T*>(static_cast<char*>(ws) + off);
}

// ---- launch helpers ----------------------------------------------------------

void fill_common(GemmParams& p, const Alg& a, int64_t M, int elem, const int32_t* perm,
                 const int32_t* offsets) {
  std::memset(&p, 0, sizeof(p));
  p.q = a.q;
  p.law = a.law;
  p.M = static_cast<int32_t>(M);
  p.K = static_cast<int32_t>(a.K());
  p.N = static_cast<int32_t>(a.N());
  p.elem = elem;
  p.perm = perm;
  p.offsets = offsets;
  for (int g = 0; g <= a.q; ++g) {
    p.S[g] = static_cast<int32_t>(a.S[g]);
    p.R[g] = static_cast<int32_t>(a.R[g]);
  }
  for (int g = 0; g < kMaxQGroups; ++g) {
    p.adj[g] = a.adj[g];
    p.adj_in[g] = a.adj_in[g];
  }
  p.nsplit = 1;
}

// the law and group widths of a parameter block, for host-side tile choices
Alg alg_of(const GemmParams& p) {
  Alg a;
  a.q = p.q;
  a.law = p.law;
  for (int g = 0; g <= p.q; ++g) {
    a.S[g] = p.S[g];
    a.R[g] = p.R[g];
  }
  return a;
}

// column-tile prefix over groups of widths given by starts G
void fill_tiles(int32_t* pfx, const int64_t* G, int q, int tile) {
  pfx[0] = 0;
  for (int g = 0; g < q; ++g) pfx[g + 1] = pfx[g] + tiles_of(G[g + 1] - G[g], tile);
}

// One workgroup per CU at most (each uses 96-128 KB of LDS); a multiple of
// 8 so that every XCD gets the same number of workgroups.
int persistent_grid(int64_t upper_tiles) {
  const int64_t cap = static_cast<int64_t>(cu_count());
  int64_t g = std::min<int64_t>(std::max<int64_t>(upper_tiles, 1), cap);
  g = (g + 7) / 8 * 8;
  return static_cast<int>(g);
}

// Column-tile width of the fp32 kernel's forward and activation-gradient
// tiles: 128 columns.
constexpr int kFp32NW = 2;

star_status hip_status(hipError_t e) { return e == hipSuccess ? STAR_OK : STAR_ERR_HIP; }

// bf16 operands take the kernel fed by direct global-to-LDS copies (its
// column tiles are wider, so the tile counts are redone for it); fp32
// operands the register-staged one.  `upper` bounds the number of tiles of
// the register-staged kernel.
// The forward takes the small-tile kernel (64 rows x 128 columns) when the
// wide kernel's 256 x 256 tiles would be at most three quarters full (rows
// taken as spread evenly over the types; a group's last column tile counts
// its empty columns) or too few to fill the chip, and when an input group is
// narrower than 64 (a 64-wide K step would span groups).  The bar was set
// by timing both kernels on the projection shapes of the paper's kernel
// study (M = 512, 2048, 8192; q = 4 to 64).
std::atomic<int> g_fwd_tiles{STAR_TILES_AUTO};

bool use_narrow_fwd(const GemmParams& p) {
  if (p.elem != 1) return false;
  for (int g = 0; g < p.q; ++g)
    if (p.S[g + 1] - p.S[g] < 64) return true;
  const int forced = g_fwd_tiles.load(std::memory_order_relaxed);
  if (forced != STAR_TILES_AUTO) return forced == STAR_TILES_SMALL;
  if (static_cast<int64_t>(p.M) < p.q) return true;
  const double m = static_cast<double>(p.M) / p.q;  // rows per type
  const double row_tiles = std::ceil(m / 256.0);
  double cols = 0.0, col_tiles = 0.0;
  for (int g = 0; g < p.q; ++g) {
    const int w = p.R[g + 1] - p.R[g];
    cols += w;
    col_tiles += (w + 255) / 256;
  }
  if (col_tiles == 0.0) return true;
  const double fill = (m / (256.0 * row_tiles)) * (cols / (256.0 * col_tiles));
  // A tile's mean contraction: K for the dense law, about two groups' worth
  // otherwise.  Over 1024 or more features the 256 x 256 tiles run their
  // MFMAs at a higher rate than the small tiles lose to padding (measured:
  // 16384 rows, 3072 -> 768 at q = 2, three quarters filled, is 30 % faster
  // on them).
  const double kc = p.law == STAR_LAW_DENSE ? p.K : std::min<double>(p.K, 2.0 * p.K / p.q);
  return (fill <= 0.75 && kc < 1024.0) || p.q * row_tiles * col_tiles < 128.0;
}

// The small-tile forward: column tiles per output group, then the launch.
hipError_t launch_narrow(NarrowParams& pn, hipStream_t stream) {
  const int tn = gemm_narrow_cols();
  pn.NTp[0] = 0;
  for (int g = 0; g < pn.q; ++g) pn.NTp[g + 1] = pn.NTp[g] + (pn.R[g + 1] - pn.R[g] + tn - 1) / tn;
  return launch_gemm_narrow(pn, gemm_narrow_row_blocks_upper(pn.M, pn.q), pn.NTp[pn.q], cu_count(), stream);
}

hipError_t launch_proj_gemm(int mode, const GemmParams& p, int nw, int64_t upper,
                            hipStream_t stream) {
  if (mode == kModeFwd && use_narrow_fwd(p)) {
    NarrowParams pn;
    std::memset(&pn, 0, sizeof(pn));
    pn.q = p.q;
    pn.law = p.law;
    pn.M = p.M;
    pn.K = p.K;
    pn.N = p.N;
    pn.act = p.act;
    pn.ydtype = p.ydtype;
    pn.perm = p.perm;
    pn.offsets = p.offsets;
    pn.A = p.A;
    pn.B = p.B;
    pn.bias = p.bias;
    pn.Z = p.Z;
    pn.Y = p.Y;
    for (int g = 0; g <= p.q; ++g) {
      pn.S[g] = p.S[g];
      pn.R[g] = p.R[g];
    }
    for (int g = 0; g < kMaxQGroups; ++g) pn.adj[g] = p.adj[g];
    return launch_narrow(pn, stream);
  }
  if (p.elem == 1) {
    GemmParams pa = p;
    const int32_t* G = (mode == kModeFwd) ? p.R : p.S;  // output column groups
    int tn = async_tile_n(alg_of(p), mode, p.M, p.act != STAR_ACT_NONE);
    pa.tile_m = kTileM;
    if (mode == kModeFwd) {
      const int forced = g_fwd_tiles.load(std::memory_order_relaxed);
      if (forced == STAR_TILES_WIDE) tn = 256;
      if (forced == STAR_TILES_WIDE192) tn = p.law == STAR_LAW_STAR || p.law == STAR_LAW_DENSE ? 192 : 256;
    }
    pa.tile_n = tn;
    pa.NTp[0] = 0;
    for (int g = 0; g < p.q; ++g) pa.NTp[g + 1] = pa.NTp[g] + (G[g + 1] - G[g] + tn - 1) / tn;
    const int64_t rows_upper = static_cast<int64_t>(p.M) / kTileM + p.q;
    return launch_gemm_async(mode, pa, rows_upper * pa.NTp[p.q], cu_count(), stream);
  }
  return launch_gemm(mode, p, nw, persistent_grid(upper), stream);
}

star_status run_plan(const int32_t* row_type, int64_t M, int q, void* ws, const PlanWs& pw,
                     hipStream_t stream) {
  return hip_status(launch_type_plan(row_type, M, q, at<int32_t>(ws, pw.perm),
                                     at<int32_t>(ws, pw.offsets), stream));
}

star_status run_fwd(const Alg& a, int64_t M, const int32_t* perm, const int32_t* offsets,
                    const void* X, const void* W, int elem, const float* bias, star_act act,
                    void* Z, void* Y, star_dtype yt, hipStream_t stream) {
  if (a.q > kMaxQGroups) {  // more groups than the other kernels take: the small tiles
    NarrowParams pn;
    std::memset(&pn, 0, sizeof(pn));
    pn.q = a.q;
    pn.law = a.law;
    pn.M = static_cast<int32_t>(M);
    pn.K = static_cast<int32_t>(a.K());
    pn.N = static_cast<int32_t>(a.N());
    pn.act = act;
    pn.ydtype = yt;
    pn.perm = perm;
    pn.offsets = offsets;
    pn.A = X;
    pn.B = W;
    pn.bias = bias;
    pn.Z = Z;
    pn.Y = Y;
    for (int g = 0; g <= a.q; ++g) {
      pn.S[g] = static_cast<int32_t>(a.S[g]);
      pn.R[g] = static_cast<int32_t>(a.R[g]);
    }
    return hip_status(launch_narrow(pn, stream));
  }
  GemmParams p;
  fill_common(p, a, M, elem, perm, offsets);
  p.A = X;
  p.B = W;
  p.bias = bias;
  p.act = act;
  p.Z = Z;
  p.Y = Y;
  p.ydtype = yt;
  const int64_t rows_upper = M / kTileM + a.q;
  const int nw = kFp32NW;
  fill_tiles(p.NTp, a.R, a.q, 64 * nw);
  const int64_t upper = rows_upper * static_cast<int64_t>(p.NTp[a.q]);
  star_status st = hip_status(launch_proj_gemm(kModeFwd, p, nw, upper, stream));
  // graph law: the output groups that are not slots of a row's type
  if (st == STAR_OK && a.law == STAR_LAW_GRAPH) st = hip_status(launch_graph_fill(kModeFwd, p, stream));
  return st;
}

star_status check_common(const star_algebra* alg, int64_t M, const int32_t* row_type, Alg& a,
                         bool large = false) {
  star_status st = parse_alg(alg, a, large);
  if (st != STAR_OK) return st;
  if (M < 0 || M > kMaxDim) return STAR_ERR_SHAPE;
  if (M > 0 && !row_type) return STAR_ERR_ARG;
  if (row_type && !aligned4(row_type)) return STAR_ERR_ALIGN;
  return STAR_OK;
}

}  // namespace

extern "C" {

const char* star_status_string(star_status s) {
  switch (s) {
    case STAR_OK: return "ok";
    case STAR_ERR_ARG: return "invalid argument";
    case STAR_ERR_SHAPE: return "invalid shape";
    case STAR_ERR_DTYPE: return "unsupported dtype combination";
    case STAR_ERR_ALIGN: return "misaligned pointer or width";
    case STAR_ERR_WORKSPACE: return "workspace missing or too small";
    case STAR_ERR_UNSUPPORTED: return "unsupported configuration";
    case STAR_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

size_t star_workspace_bytes(int32_t op, const star_algebra* alg, const star_algebra* alg2,
                            int64_t M) {
  Alg a;
  if (parse_alg(alg, a, op == STAR_OP_FWD) != STAR_OK || M < 0) return 0;
  switch (op) {
    case STAR_OP_FWD:
    case STAR_OP_BWD_DATA:
    case STAR_OP_FFN_FWD:
      return plan_layout(M, a.q).end;
    case STAR_OP_BWD_WEIGHT:
      return bwd_weight_layout(a, M).end;
    case STAR_OP_DECODE: {
      Alg d;
      if (parse_alg(alg2, d) != STAR_OK) return 0;
      const int64_t m = std::min<int64_t>(M, kDecodeMaxRows);
      // the single-launch stack's layout only where the stack can run
      const StackPlan sp = stack_plan(a, d, std::max<int64_t>(m, 1), 1);
      return sp.ok ? std::max(decode_layout(a, m).end, sp.end) : decode_layout(a, m).end;
    }
    default:
      return 0;
  }
}

int star_set_fwd_tiles(int tiles) {
  if (tiles != STAR_TILES_AUTO && tiles != STAR_TILES_WIDE && tiles != STAR_TILES_SMALL &&
      tiles != STAR_TILES_WIDE192)
    return -1;
  return g_fwd_tiles.exchange(tiles);
}

star_status star_count_products(const star_algebra* alg, int64_t* per_type) {
  Alg a;
  star_status st = parse_alg(alg, a, true);
  if (st != STAR_OK) return st;
  if (!per_type) return STAR_ERR_ARG;
  for (int i = 0; i < a.q; ++i) {
    int64_t n = 0;
    for (int j = 0; j < a.q; ++j)
      for (int k = 0; k < a.q; ++k) n += host_in_support(a, i, j, k) ? 1 : 0;
    per_type[i] = n;
  }
  return STAR_OK;
}

star_status star_count_macs(const star_algebra* alg, const int64_t* rows_per_type, int64_t* macs) {
  Alg a;
  star_status st = parse_alg(alg, a, true);
  if (st != STAR_OK) return st;
  if (!rows_per_type || !macs) return STAR_ERR_ARG;
  int64_t total = 0;
  for (int i = 0; i < a.q; ++i) {
    int64_t row = 0;
    for (int j = 0; j < a.q; ++j)
      for (int k = 0; k < a.q; ++k)
        if (host_in_support(a, i, j, k)) row += a.s(k) * a.r(j);
    total += rows_per_type[i] * row;
  }
  *macs = total;
  return STAR_OK;
}

size_t star_plan_bytes(int32_t q, int64_t M) {
  if (q < 1 || q > kMaxQFwd || M < 0 || M > kMaxDim) return 0;
  return plan_layout(M, q).end;
}

star_status star_type_plan(int32_t q, int64_t M, const int32_t* row_type, void* plan,
                           size_t plan_bytes, hipStream_t stream) {
  if (q < 1 || q > kMaxQFwd) return STAR_ERR_ARG;
  if (M < 0 || M > kMaxDim) return STAR_ERR_SHAPE;
  if (M == 0) return STAR_OK;
  if (!row_type || !plan) return STAR_ERR_ARG;
  if (!aligned4(row_type) || !aligned16(plan)) return STAR_ERR_ALIGN;
  const PlanWs pw = plan_layout(M, q);
  if (plan_bytes < pw.end) return STAR_ERR_WORKSPACE;
  return run_plan(row_type, M, q, plan, pw, stream);
}

// The *_planned entry points take a plan built by star_type_plan; the
// plain entry points build it into the head of their workspace first.

star_status star_proj_fwd_planned(const star_algebra* alg, int64_t M, const void* plan,
                                  const void* X, star_dtype xt, const void* W, star_dtype wt,
                                  const float* bias, star_act act, void* Z_out, void* Y,
                                  star_dtype yt, hipStream_t stream) {
  Alg a;
  star_status st = parse_alg(alg, a, true);
  if (st != STAR_OK) return st;
  if (M < 0 || M > kMaxDim) return STAR_ERR_SHAPE;
  if (!valid_dtype(xt) || !valid_dtype(wt) || !valid_dtype(yt) || xt != wt) return STAR_ERR_DTYPE;
  if (a.q > kMaxQGroups && xt != STAR_BF16) return STAR_ERR_UNSUPPORTED;
  if (!valid_act(act)) return STAR_ERR_ARG;
  if (M == 0) return STAR_OK;
  if (!plan || !X || !W || !Y) return STAR_ERR_ARG;
  if (!aligned16(plan) || !aligned16(X) || !aligned16(W) || !aligned16(Y) ||
      (Z_out && !aligned16(Z_out)) || (bias && !aligned16(bias)))
    return STAR_ERR_ALIGN;
  const PlanWs pw = plan_layout(M, a.q);
  void* pl = const_cast<void*>(plan);
  return run_fwd(a, M, at<int32_t>(pl, pw.perm), at<int32_t>(pl, pw.offsets), X, W,
                 xt == STAR_BF16 ? 1 : 0, bias, act, Z_out, Y, yt, stream);
}

star_status star_proj_fwd(const star_algebra* alg, int64_t M, const int32_t* row_type,
                          const void* X, star_dtype xt, const void* W, star_dtype wt,
                          const float* bias, star_act act, void* Z_out, void* Y, star_dtype yt,
                          void* ws, size_t ws_bytes, hipStream_t stream) {
  Alg a;
  star_status st = check_common(alg, M, row_type, a, true);
  if (st != STAR_OK) return st;
  if (!valid_dtype(xt) || !valid_dtype(wt) || !valid_dtype(yt) || xt != wt) return STAR_ERR_DTYPE;
  if (a.q > kMaxQGroups && xt != STAR_BF16) return STAR_ERR_UNSUPPORTED;
  if (!valid_act(act)) return STAR_ERR_ARG;
  if (M == 0) return STAR_OK;
  if (!X || !W || !Y) return STAR_ERR_ARG;
  if (!aligned16(X) || !aligned16(W) || !aligned16(Y) || (Z_out && !aligned16(Z_out)) ||
      (bias && !aligned16(bias)))
    return STAR_ERR_ALIGN;
  const PlanWs pw = plan_layout(M, a.q);
  if (!ws || ws_bytes < pw.end) return STAR_ERR_WORKSPACE;
  if (!aligned16(ws)) return STAR_ERR_ALIGN;
  st = run_plan(row_type, M, a.q, ws, pw, stream);
  if (st != STAR_OK) return st;
  return star_proj_fwd_planned(alg, M, ws, X, xt, W, wt, bias, act, Z_out, Y, yt, stream);
}

star_status star_proj_bwd_data_planned(const star_algebra* alg, int64_t M, const void* plan,
                                       const void* dY, star_dtype dyt, const void* W,
                                       star_dtype wt, const void* Z_prev, star_act act_prev,
                                       void* dX, star_dtype dxt, hipStream_t stream) {
  Alg a;
  star_status st = parse_alg(alg, a);
  if (st != STAR_OK) return st;
  if (M < 0 || M > kMaxDim) return STAR_ERR_SHAPE;
  if (!valid_dtype(dyt) || !valid_dtype(wt) || !valid_dtype(dxt) || dyt != wt)
    return STAR_ERR_DTYPE;
  if (!valid_act(act_prev)) return STAR_ERR_ARG;
  if (M == 0) return STAR_OK;
  if (!plan || !dY || !W || !dX) return STAR_ERR_ARG;
  if (!aligned16(plan) || !aligned16(dY) || !aligned16(W) || !aligned16(dX) ||
      (Z_prev && !aligned16(Z_prev)))
    return STAR_ERR_ALIGN;
  const PlanWs pw = plan_layout(M, a.q);
  void* pl = const_cast<void*>(plan);
  GemmParams p;
  fill_common(p, a, M, dyt == STAR_BF16 ? 1 : 0, at<int32_t>(pl, pw.perm),
              at<int32_t>(pl, pw.offsets));
  p.A = dY;
  p.B = W;
  p.Zprev = Z_prev;
  p.act = Z_prev ? act_prev : STAR_ACT_NONE;
  p.Y = dX;
  p.ydtype = dxt;
  const int64_t rows_upper = M / kTileM + a.q;
  const int nw = kFp32NW;
  fill_tiles(p.NTp, a.S, a.q, 64 * nw);
  const int64_t upper = rows_upper * static_cast<int64_t>(p.NTp[a.q]);
  st = hip_status(launch_proj_gemm(kModeBwdData, p, nw, upper, stream));
  // graph law: zero gradient for the input groups that are not slots
  if (st == STAR_OK && a.law == STAR_LAW_GRAPH) st = hip_status(launch_graph_fill(kModeBwdData, p, stream));
  return st;
}

star_status star_proj_bwd_data(const star_algebra* alg, int64_t M, const int32_t* row_type,
                               const void* dY, star_dtype dyt, const void* W, star_dtype wt,
                               const void* Z_prev, star_act act_prev, void* dX, star_dtype dxt,
                               void* ws, size_t ws_bytes, hipStream_t stream) {
  Alg a;
  star_status st = check_common(alg, M, row_type, a);
  if (st != STAR_OK) return st;
  if (!valid_dtype(dyt) || !valid_dtype(wt) || !valid_dtype(dxt) || dyt != wt)
    return STAR_ERR_DTYPE;
  if (!valid_act(act_prev)) return STAR_ERR_ARG;
  if (M == 0) return STAR_OK;
  if (!dY || !W || !dX) return STAR_ERR_ARG;
  if (!aligned16(dY) || !aligned16(W) || !aligned16(dX) || (Z_prev && !aligned16(Z_prev)))
    return STAR_ERR_ALIGN;
  const PlanWs pw = plan_layout(M, a.q);
  if (!ws || ws_bytes < pw.end) return STAR_ERR_WORKSPACE;
  if (!aligned16(ws)) return STAR_ERR_ALIGN;
  st = run_plan(row_type, M, a.q, ws, pw, stream);
  if (st != STAR_OK) return st;
  return star_proj_bwd_data_planned(alg, M, ws, dY, dyt, W, wt, Z_prev, act_prev, dX, dxt,
                                    stream);
}

star_status star_proj_bwd_weight_planned(const star_algebra* alg, int64_t M, const void* plan,
                                         const void* X, star_dtype xt, const void* dY,
                                         star_dtype dyt, float* dW, float* dbias, void* ws,
                                         size_t ws_bytes, hipStream_t stream) {
  Alg a;
  star_status st = parse_alg(alg, a);
  if (st != STAR_OK) return st;
  if (M < 0 || M > kMaxDim) return STAR_ERR_SHAPE;
  if (!valid_dtype(xt) || !valid_dtype(dyt) || xt != dyt) return STAR_ERR_DTYPE;
  if (!dW) return STAR_ERR_ARG;
  if (M > 0 && (!X || !dY || !plan)) return STAR_ERR_ARG;
  if ((X && !aligned16(X)) || (dY && !aligned16(dY)) || !aligned16(dW) ||
      (dbias && !aligned4(dbias)) || (plan && !aligned16(plan)))
    return STAR_ERR_ALIGN;
  const BwdWs bw = bwd_weight_layout(a, M);
  const bool pipelined = xt == STAR_BF16;
  const bool need_ws = pipelined || bw.nsplit > 1 || (a.law == STAR_LAW_GRAPH && dbias);
  if (need_ws && M > 0 && (!ws || ws_bytes < bw.end)) return STAR_ERR_WORKSPACE;
  if (ws && !aligned16(ws)) return STAR_ERR_ALIGN;
  // M = 0 still defines the output: an empty sum
  if (M == 0) {
    hipError_t e = launch_fill_zero(dW, a.K() * a.N(), stream);
    if (e == hipSuccess && dbias) e = launch_fill_zero(dbias, a.N(), stream);
    return hip_status(e);
  }
  const PlanWs pw = plan_layout(M, a.q);
  void* pl = const_cast<void*>(plan);
  GemmParams p;
  fill_common(p, a, M, xt == STAR_BF16 ? 1 : 0, at<int32_t>(pl, pw.perm),
              at<int32_t>(pl, pw.offsets));
  if (pipelined) {
    // every tile contracts over a range of type-sorted positions; the
    // kernel reads the rows of X and dY at those positions through perm
    const TileShape ts = async_tiles_weight(a, M);
    p.tile_m = ts.tm;
    p.tile_n = ts.tn;
    fill_tiles(p.NTp, a.R, a.q, p.tile_n);
    fill_tiles(p.MTp, a.S, a.q, p.tile_m);
    p.A = X;
    p.B = dY;
    p.dW = dW;
    p.nsplit = bw.nsplit_a;
    if (bw.nsplit_a > 1) p.partial = at<float>(ws, bw.partial_a);
    const int64_t upper = static_cast<int64_t>(p.MTp[a.q]) * p.NTp[a.q] * p.nsplit;
    st = hip_status(launch_gemm_async(kModeBwdWeight, p, upper, cu_count(), stream));
    if (st == STAR_OK && bw.nsplit_a > 1)
      st = hip_status(launch_sum_partials(p.partial, p.nsplit, static_cast<int64_t>(p.K) * p.N, dW, stream));
    if (st != STAR_OK || !dbias) return st;
    // dbias = column sums of dY over the rows of valid type, in fixed chunks
    const int32_t chunk = static_cast<int32_t>((M + kColSumChunks - 1) / kColSumChunks);
    float* cs = at<float>(ws, bw.colsum);
    st = hip_status(launch_column_sum(static_cast<const uint16_t*>(dY), p.N, p.perm, p.offsets, a.q, p.M,
                                      chunk, kColSumChunks, cs, stream));
    if (st != STAR_OK) return st;
    return hip_status(launch_sum_chunks(cs, kColSumChunks, p.N, dbias, stream));
  }
  fill_tiles(p.NTp, a.R, a.q, 64 * kBwdWeightNW);
  fill_tiles(p.MTp, a.S, a.q, kTileM);
  p.A = X;
  p.B = dY;
  p.dW = dW;
  // the graph law's diagonal tiles do not contract over every row, so its
  // bias gradient is summed apart (below)
  p.dbias = a.law == STAR_LAW_GRAPH ? nullptr : dbias;
  p.nsplit = bw.nsplit;
  if (bw.nsplit > 1) {
    p.partial = at<float>(ws, bw.partial);
    p.dbias_part = at<float>(ws, bw.dbias_part);
  }
  const int64_t upper = static_cast<int64_t>(p.MTp[a.q]) * p.NTp[a.q] * p.nsplit;
  st = hip_status(launch_gemm(kModeBwdWeight, p, kBwdWeightNW, persistent_grid(upper), stream));
  if (st == STAR_OK && bw.nsplit > 1) st = hip_status(launch_split_reduce(p, stream));
  if (st != STAR_OK || a.law != STAR_LAW_GRAPH || !dbias) return st;
  const int32_t chunk = static_cast<int32_t>((M + kColSumChunks - 1) / kColSumChunks);
  float* cs = at<float>(ws, bw.colsum);
  st = hip_status(launch_column_sum_f32(static_cast<const float*>(dY), p.N, p.perm, p.offsets, a.q, p.M, chunk,
                                        kColSumChunks, cs, stream));
  if (st != STAR_OK) return st;
  return hip_status(launch_sum_chunks(cs, kColSumChunks, p.N, dbias, stream));
}

star_status star_proj_bwd_weight(const star_algebra* alg, int64_t M, const int32_t* row_type,
                                 const void* X, star_dtype xt, const void* dY, star_dtype dyt,
                                 float* dW, float* dbias, void* ws, size_t ws_bytes,
                                 hipStream_t stream) {
  Alg a;
  star_status st = check_common(alg, M, row_type, a);
  if (st != STAR_OK) return st;
  if (!valid_dtype(xt) || !valid_dtype(dyt) || xt != dyt) return STAR_ERR_DTYPE;
  if (!dW) return STAR_ERR_ARG;
  if (M > 0 && (!X || !dY)) return STAR_ERR_ARG;
  if ((X && !aligned16(X)) || (dY && !aligned16(dY)) || !aligned16(dW) ||
      (dbias && !aligned4(dbias)))
    return STAR_ERR_ALIGN;
  const BwdWs bw = bwd_weight_layout(a, M);
  if (!ws || ws_bytes < bw.end) return STAR_ERR_WORKSPACE;
  if (!aligned16(ws)) return STAR_ERR_ALIGN;
  if (M > 0) {
    st = run_plan(row_type, M, a.q, ws, bw.plan, stream);
    if (st != STAR_OK) return st;
  }
  return star_proj_bwd_weight_planned(alg, M, ws, X, xt, dY, dyt, dW, dbias, ws, ws_bytes,
                                      stream);
}

star_status star_ffn_fwd(const star_algebra* up, const star_algebra* down, int64_t M,
                         const int32_t* row_type, const void* X, const void* W_up,
                         const float* b_up, const void* W_down, const float* b_down,
                         star_act act, void* Z_up, void* H, void* Y, star_dtype dt,
                         star_dtype yt, void* ws, size_t ws_bytes, hipStream_t stream) {
  Alg u, d;
  star_status st = check_common(up, M, row_type, u);
  if (st != STAR_OK) return st;
  st = parse_alg(down, d);
  if (st != STAR_OK) return st;
  if (d.q != u.q) return STAR_ERR_SHAPE;
  for (int g = 0; g < u.q; ++g)
    if (d.s(g) != u.r(g)) return STAR_ERR_SHAPE;
  if (!valid_dtype(dt) || !valid_dtype(yt)) return STAR_ERR_DTYPE;
  if (!valid_act(act)) return STAR_ERR_ARG;
  if (M == 0) return STAR_OK;
  if (!X || !W_up || !W_down || !H || !Y) return STAR_ERR_ARG;
  if (!aligned16(X) || !aligned16(W_up) || !aligned16(W_down) || !aligned16(H) ||
      !aligned16(Y) || (Z_up && !aligned16(Z_up)) || (b_up && !aligned16(b_up)) ||
      (b_down && !aligned16(b_down)))
    return STAR_ERR_ALIGN;
  const PlanWs pw = plan_layout(M, u.q);
  if (!ws || ws_bytes < pw.end) return STAR_ERR_WORKSPACE;
  if (!aligned16(ws)) return STAR_ERR_ALIGN;
  st = run_plan(row_type, M, u.q, ws, pw, stream);
  if (st != STAR_OK) return st;
  const int elem = dt == STAR_BF16 ? 1 : 0;
  const int32_t* perm = at<int32_t>(ws, pw.perm);
  const int32_t* offs = at<int32_t>(ws, pw.offsets);
  st = run_fwd(u, M, perm, offs, X, W_up, elem, b_up, act, Z_up, H, dt, stream);
  if (st != STAR_OK) return st;
  return run_fwd(d, M, perm, offs, H, W_down, elem, b_down, STAR_ACT_NONE, nullptr, Y, yt, stream);
}

}  // extern "C"

namespace {
// The decode step behind star_decode and star_decode_gated (W_gate non-null:
// gated FFN, persistent stack only).
star_status decode_impl(const star_algebra* up, const star_algebra* down, int32_t n_layers, int64_t M,
                        const int32_t* row_type, const void* X, star_dtype xt, const void* const* W_gate,
                        const float* const* b_gate, const void* const* W_up, const float* const* b_up,
                        const void* const* W_down, const float* const* b_down, star_act act,
                        int32_t residual, void* Y, star_dtype yt, void* ws, size_t ws_bytes,
                        hipStream_t stream, int32_t* err_word = nullptr) {
  const bool gated = W_gate != nullptr;
  Alg u, d;
  star_status st = check_common(up, M, row_type, u);
  if (st != STAR_OK) return st;
  st = parse_alg(down, d);
  if (st != STAR_OK) return st;
  if (d.K() != u.N() || d.N() != u.K()) return STAR_ERR_SHAPE;
  if (M > kDecodeMaxRows || u.K() > kDecodeMaxK || u.N() > kDecodeMaxK) return STAR_ERR_UNSUPPORTED;
  if (n_layers < 1) return STAR_ERR_ARG;
  if (!valid_dtype(yt) || xt != STAR_BF16) return STAR_ERR_DTYPE;
  if (!valid_act(act)) return STAR_ERR_ARG;
  if (M == 0) return STAR_OK;
  if (!X || !W_up || !W_down || !Y) return STAR_ERR_ARG;
  if (!aligned16(X) || !aligned16(Y)) return STAR_ERR_ALIGN;
  for (int l = 0; l < n_layers; ++l) {
    if (!W_up[l] || !W_down[l] || (gated && !W_gate[l])) return STAR_ERR_ARG;
    if (!aligned16(W_up[l]) || !aligned16(W_down[l]) || (gated && !aligned16(W_gate[l]))) return STAR_ERR_ALIGN;
    if ((b_up && b_up[l] && !aligned16(b_up[l])) || (b_down && b_down[l] && !aligned16(b_down[l])) ||
        (gated && b_gate && b_gate[l] && !aligned16(b_gate[l])))
      return STAR_ERR_ALIGN;
  }
  const DecodeWs dw = decode_layout(u, M);
  const StackPlan sp = stack_plan(u, d, M, n_layers, gated);
  if (!ws || ws_bytes < (sp.ok ? std::max(dw.end, sp.end) : dw.end)) return STAR_ERR_WORKSPACE;
  if (!aligned16(ws)) return STAR_ERR_ALIGN;
  // the gated FFN runs only in the persistent stack
  if (gated && !sp.ok) return STAR_ERR_UNSUPPORTED;
  // the error flag: the workspace's status line unless the caller gives a
  // word of its own; zeroed before anything runs
  int32_t* err = err_word ? err_word : at<int32_t>(ws, 0);
  if (err_word) {
    st = hip_status(launch_fill_zero(reinterpret_cast<float*>(err_word), 1, stream));
    if (st != STAR_OK) return st;
  }

  if (sp.ok) {
    DecodeStack k;
    std::memset(&k, 0, sizeof(k));
    k.q = u.q;
    k.law = u.law;
    k.M = static_cast<int32_t>(M);
    k.D = static_cast<int32_t>(u.K());
    k.F = static_cast<int32_t>(u.N());
    k.L = n_layers;
    k.act = act;
    k.residual = residual;
    k.ydtype = yt;
    k.ns = sp.ns;
    k.kc = sp.kc;
    k.nt_up = sp.nt_up;
    k.nt_dn = sp.nt_dn;
    for (int g = 0; g <= u.q; ++g) {
      k.SD[g] = static_cast<int32_t>(u.S[g]);
      k.SF[g] = static_cast<int32_t>(u.R[g]);
    }
    fill_tiles(k.NTu, u.R, u.q, kDecodeTileN);
    fill_tiles(k.NTd, d.R, d.q, kDecodeTileN);
    k.types = row_type;
    for (int g = 0; g < kMaxQGroups; ++g) k.adj[g] = u.adj[g];
    k.X = static_cast<const uint16_t*>(X);
    for (int l = 0; l < n_layers; ++l) {
      k.Wu[l] = static_cast<const uint16_t*>(W_up[l]);
      k.Wd[l] = static_cast<const uint16_t*>(W_down[l]);
      k.bu[l] = b_up ? b_up[l] : nullptr;
      k.bd[l] = b_down ? b_down[l] : nullptr;
      if (gated) {
        k.Wg[l] = static_cast<const uint16_t*>(W_gate[l]);
        k.bg[l] = b_gate ? b_gate[l] : nullptr;
      }
    }
    k.gated = gated ? 1 : 0;
    k.Y = Y;
    k.H = at<uint16_t>(ws, sp.H);
    k.hb = at<uint16_t>(ws, sp.hb);
    k.h = at<float>(ws, sp.h);
    k.part = at<float>(ws, sp.part);
    k.cnt = at<int32_t>(ws, sp.cnt);
    k.err = err;
    k.tH = sp.resident ? at<uint64_t>(ws, sp.tH) : nullptr;
    k.tpart = sp.resident ? at<uint64_t>(ws, sp.tpart) : nullptr;
    st = hip_status(launch_fill_zero(at<float>(ws, sp.cnt),
                                     static_cast<int64_t>((sp.zero_end - sp.cnt) / sizeof(float)), stream));
    if (st != STAR_OK) return st;
    return hip_status(launch_decode_stack(k, sp.grid, stream));
  }

  // the status line reads zero: the per-projection kernels do not wait
  if (!err_word) {
    st = hip_status(launch_fill_zero(at<float>(ws, 0), kDecodeStatusBytes / sizeof(float), stream));
    if (st != STAR_OK) return st;
  }
  float* h = at<float>(ws, dw.h);
  uint16_t* xb = at<uint16_t>(ws, dw.xb);
  uint16_t* Hb = at<uint16_t>(ws, dw.H);
  auto fill = [&](DecodePhase& p, const Alg& a) {
    std::memset(&p, 0, sizeof(p));
    p.q = a.q;
    p.law = a.law;
    p.M = static_cast<int32_t>(M);
    p.K = static_cast<int32_t>(a.K());
    p.N = static_cast<int32_t>(a.N());
    for (int g = 0; g <= a.q; ++g) {
      p.S[g] = static_cast<int32_t>(a.S[g]);
      p.R[g] = static_cast<int32_t>(a.R[g]);
    }
    fill_tiles(p.NTp, a.R, a.q, kDecodeTileN);
    for (int g = 0; g < kMaxQGroups; ++g) p.adj[g] = a.adj[g];
    p.types = row_type;
    p.act = act;
    p.residual = residual;
  };
  DecodePhase pu, pd;
  fill(pu, u);
  fill(pd, d);
  pu.mode = 0;
  pu.out_bf16 = Hb;
  pd.mode = 1;
  pd.A = Hb;
  pd.ydtype = yt;
  for (int l = 0; l < n_layers; ++l) {
    const bool first = (l == 0), last = (l == n_layers - 1);
    pu.A = first ? static_cast<const uint16_t*>(X) : xb;
    pu.W = static_cast<const uint16_t*>(W_up[l]);
    pu.bias = b_up ? b_up[l] : nullptr;
    st = hip_status(launch_decode_phase(pu, stream));
    if (st != STAR_OK) return st;
    pd.W = static_cast<const uint16_t*>(W_down[l]);
    pd.bias = b_down ? b_down[l] : nullptr;
    // h_prev: X itself for the first layer, the fp32 state afterwards
    pd.h_init = first ? static_cast<const uint16_t*>(X) : nullptr;
    pd.h_in = first ? nullptr : h;
    pd.h_out = last ? nullptr : h;
    pd.out_bf16 = last ? nullptr : xb;
    pd.Y = last ? Y : nullptr;
    st = hip_status(launch_decode_phase(pd, stream));
    if (st != STAR_OK) return st;
  }
  return STAR_OK;
}
}  // namespace

extern "C" {

star_status star_decode(const star_algebra* up, const star_algebra* down, int32_t n_layers,
                        int64_t M, const int32_t* row_type, const void* X, star_dtype xt,
                        const void* const* W_up, const float* const* b_up,
                        const void* const* W_down, const float* const* b_down, star_act act,
                        int32_t residual, void* Y, star_dtype yt, void* ws, size_t ws_bytes,
                        hipStream_t stream) {
  return decode_impl(up, down, n_layers, M, row_type, X, xt, nullptr, nullptr, W_up, b_up, W_down, b_down,
                     act, residual, Y, yt, ws, ws_bytes, stream);
}

star_status star_decode_noalloc(const star_algebra* up, const star_algebra* down, int32_t n_layers,
                                int64_t M, const int32_t* row_type, const void* X, star_dtype xt,
                                const void* const* W_up, const float* const* b_up,
                                const void* const* W_down, const float* const* b_down, star_act act,
                                int32_t residual, void* Y, star_dtype yt, int32_t* status,
                                hipStream_t stream) {
  // the same host-side checks as star_decode, before the scratch is looked up
  Alg u, d;
  star_status st = check_common(up, M, row_type, u);
  if (st != STAR_OK) return st;
  st = parse_alg(down, d);
  if (st != STAR_OK) return st;
  if (M > kDecodeMaxRows || u.K() > kDecodeMaxK || u.N() > kDecodeMaxK) return STAR_ERR_UNSUPPORTED;
  if (xt != STAR_BF16 || !valid_dtype(yt)) return STAR_ERR_DTYPE;
  if (status && !aligned4(status)) return STAR_ERR_ALIGN;
  if (M == 0) return decode_impl(up, down, n_layers, M, row_type, X, xt, nullptr, nullptr, W_up, b_up, W_down,
                                 b_down, act, residual, Y, yt, nullptr, 0, stream);
  // a shape whose workspace exceeds the static scratch is refused
  if (star_workspace_bytes(STAR_OP_DECODE, up, down, M) > kDecodeScratchBytes) return STAR_ERR_WORKSPACE;
  void* scratch = nullptr;
  if (decode_scratch(&scratch) != hipSuccess) return STAR_ERR_HIP;
  return decode_impl(up, down, n_layers, M, row_type, X, xt, nullptr, nullptr, W_up, b_up, W_down, b_down, act,
                     residual, Y, yt, scratch, kDecodeScratchBytes, stream, status);
}

star_status star_decode_status(const void* ws, size_t ws_bytes, int32_t* timed_out, hipStream_t stream) {
  if (!ws || !timed_out) return STAR_ERR_ARG;
  if (ws_bytes < sizeof(int32_t)) return STAR_ERR_WORKSPACE;
  if (!aligned16(ws)) return STAR_ERR_ALIGN;
  int32_t host = 0;
  hipError_t e = hipMemcpyAsync(&host, ws, sizeof(host), hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  if (e != hipSuccess) return STAR_ERR_HIP;
  *timed_out = host != 0 ? 1 : 0;
  return STAR_OK;
}

star_status star_decode_gated(const star_algebra* up, const star_algebra* down, int32_t n_layers,
                              int64_t M, const int32_t* row_type, const void* X, star_dtype xt,
                              const void* const* W_gate, const float* const* b_gate,
                              const void* const* W_up, const float* const* b_up,
                              const void* const* W_down, const float* const* b_down,
                              int32_t residual, void* Y, star_dtype yt, void* ws, size_t ws_bytes,
                              hipStream_t stream) {
  if (M > 0 && !W_gate) return STAR_ERR_ARG;
  static const void* const no_layers[1] = {nullptr};
  return decode_impl(up, down, n_layers, M, row_type, X, xt, W_gate ? W_gate : no_layers, b_gate, W_up, b_up,
                     W_down, b_down, STAR_ACT_NONE, residual, Y, yt, ws, ws_bytes, stream);
}

star_status star_validate_types(int64_t M, const int32_t* row_type, int32_t q, int64_t* n_bad,
                                void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!n_bad || q < 1) return STAR_ERR_ARG;
  if (M < 0) return STAR_ERR_SHAPE;
  *n_bad = 0;
  if (M == 0) return STAR_OK;
  if (!row_type) return STAR_ERR_ARG;
  if (!ws || ws_bytes < 16) return STAR_ERR_WORKSPACE;
  if (!aligned16(ws)) return STAR_ERR_ALIGN;
  auto* cnt = static_cast<unsigned long long*>(ws);
  hipError_t e = hipMemsetAsync(cnt, 0, sizeof(unsigned long long), stream);
  if (e == hipSuccess) e = launch_count_bad_types(row_type, M, q, cnt, stream);
  unsigned long long host = 0;
  if (e == hipSuccess) e = hipMemcpyAsync(&host, cnt, sizeof(host), hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  if (e != hipSuccess) return STAR_ERR_HIP;
  *n_bad = static_cast<int64_t>(host);
  return STAR_OK;
}

namespace {
star_status check_elementwise(int64_t n, star_dtype dt, std::initializer_list<const void*> ptrs) {
  if (!valid_dtype(dt)) return STAR_ERR_DTYPE;
  if (n < 0 || n > kMaxDim * kMaxDim) return STAR_ERR_SHAPE;
  if (n % 8) return STAR_ERR_ALIGN;
  if (n == 0) return STAR_OK;
  for (const void* q : ptrs) {
    if (!q) return STAR_ERR_ARG;
    if (!aligned16(q)) return STAR_ERR_ALIGN;
  }
  return STAR_OK;
}
}  // namespace

star_status star_swiglu_fwd(int64_t n, const void* Z_gate, const void* Z_up, star_dtype dt, void* H,
                            hipStream_t stream) {
  star_status st = check_elementwise(n, dt, {Z_gate, Z_up, H});
  if (st != STAR_OK || n == 0) return st;
  return hip_status(launch_swiglu_fwd(n, dt == STAR_BF16 ? 1 : 0, Z_gate, Z_up, H, stream));
}

star_status star_swiglu_merged_fwd(int64_t M, int64_t F, const void* Z_gu, star_dtype dt, void* H,
                                   hipStream_t stream) {
  if (!valid_dtype(dt)) return STAR_ERR_DTYPE;
  if (M < 0 || F < 0 || M > kMaxDim || F > kMaxDim) return STAR_ERR_SHAPE;
  if (F % 8) return STAR_ERR_ALIGN;
  if (M == 0 || F == 0) return STAR_OK;
  if (!Z_gu || !H) return STAR_ERR_ARG;
  if (!aligned16(Z_gu) || !aligned16(H)) return STAR_ERR_ALIGN;
  return hip_status(launch_swiglu_merged(M, F, dt == STAR_BF16 ? 1 : 0, Z_gu, H, stream));
}

star_status star_swiglu_up_fwd_planned(const star_algebra* alg_gu, int64_t M, const void* plan, const void* X,
                                       star_dtype xt, const void* W_gu, star_dtype wt, const float* b_gu,
                                       void* Z_out, void* H, star_dtype ht, hipStream_t stream) {
  Alg a;
  star_status st = parse_alg(alg_gu, a, true);
  if (st != STAR_OK) return st;
  if (a.law == STAR_LAW_GRAPH) return STAR_ERR_UNSUPPORTED;
  for (int g = 0; g < a.q; ++g)
    if (a.r(g) % 16) return STAR_ERR_UNSUPPORTED;
  if (M < 0 || M > kMaxDim) return STAR_ERR_SHAPE;
  if (!valid_dtype(xt) || !valid_dtype(wt) || !valid_dtype(ht) || xt != wt) return STAR_ERR_DTYPE;
  if (xt != STAR_BF16) return STAR_ERR_UNSUPPORTED;
  if (M == 0) return STAR_OK;
  if (!plan || !X || !W_gu || !H) return STAR_ERR_ARG;
  if (!aligned16(plan) || !aligned16(X) || !aligned16(W_gu) || !aligned16(H) || (Z_out && !aligned16(Z_out)) ||
      (b_gu && !aligned16(b_gu)))
    return STAR_ERR_ALIGN;
  const PlanWs pw = plan_layout(M, a.q);
  void* pl = const_cast<void*>(plan);
  NarrowParams pn;
  std::memset(&pn, 0, sizeof(pn));
  pn.q = a.q;
  pn.law = a.law;
  pn.M = static_cast<int32_t>(M);
  pn.K = static_cast<int32_t>(a.K());
  pn.N = static_cast<int32_t>(a.N());
  pn.act = STAR_ACT_NONE;
  pn.ydtype = ht;
  pn.swiglu = 1;
  pn.perm = at<int32_t>(pl, pw.perm);
  pn.offsets = at<int32_t>(pl, pw.offsets);
  pn.A = X;
  pn.B = W_gu;
  pn.bias = b_gu;
  pn.Z = Z_out;
  pn.Y = H;
  for (int g = 0; g <= a.q; ++g) {
    pn.S[g] = static_cast<int32_t>(a.S[g]);
    pn.R[g] = static_cast<int32_t>(a.R[g]);
  }
  return hip_status(launch_narrow(pn, stream));
}

star_status star_swiglu_bwd(int64_t n, const void* dH, const void* Z_gate, const void* Z_up, star_dtype dt,
                            void* dZ_gate, void* dZ_up, hipStream_t stream) {
  star_status st = check_elementwise(n, dt, {dH, Z_gate, Z_up, dZ_gate, dZ_up});
  if (st != STAR_OK || n == 0) return st;
  return hip_status(launch_swiglu_bwd(n, dt == STAR_BF16 ? 1 : 0, dH, Z_gate, Z_up, dZ_gate, dZ_up, stream));
}

star_status star_add(int64_t n, const void* a, const void* b, star_dtype dt, void* out, hipStream_t stream) {
  star_status st = check_elementwise(n, dt, {a, b, out});
  if (st != STAR_OK || n == 0) return st;
  return hip_status(launch_add(n, dt == STAR_BF16 ? 1 : 0, a, b, out, stream));
}

// ---- algebraic attention --------------------------------------------------

// (helpers: C++ linkage inside the C-linkage block)
extern "C++" {
namespace {
struct AttnShape {
  int32_t B, S, H, Hkv, D, q, law;
};
star_status parse_attn(const star_attn_shape* sh, AttnShape& a) {
  if (!sh) return STAR_ERR_ARG;
  if (sh->law != STAR_LAW_STAR && sh->law != STAR_LAW_DENSE && sh->law != STAR_LAW_TENSOR2) {
    return sh->law == STAR_LAW_GRAPH ? STAR_ERR_UNSUPPORTED : STAR_ERR_ARG;
  }
  if (sh->batch < 0 || sh->seq_len < 0 || sh->n_heads < 1 || sh->n_kv_heads < 1) return STAR_ERR_SHAPE;
  if (sh->n_heads % sh->n_kv_heads) return STAR_ERR_SHAPE;
  if (sh->head_dim != 64 && sh->head_dim != 128) return STAR_ERR_UNSUPPORTED;
  if (sh->q < 1 || sh->head_dim % sh->q || (sh->head_dim / sh->q) % 8) return STAR_ERR_UNSUPPORTED;
  if (sh->law == STAR_LAW_TENSOR2 && sh->q != 1 && sh->q != 2 && sh->q != 4) return STAR_ERR_UNSUPPORTED;
  if (sh->seq_len > (1 << 30)) return STAR_ERR_SHAPE;
  a = {sh->batch, sh->seq_len, sh->n_heads, sh->n_kv_heads, sh->head_dim, sh->q, sh->law};
  return STAR_OK;
}
AttnParams attn_params(const AttnShape& a) {
  AttnParams p{};
  p.B = a.B;
  p.S = a.S;
  p.n_heads = a.H;
  p.n_kv = a.Hkv;
  p.head_dim = a.D;
  p.q = a.q;
  p.law = a.law;
  return p;
}
struct AttnDecWs {
  int32_t chunk = 0, nchunks = 0;
  size_t part_o = 0, part_ml = 0, end = 0;
};
AttnDecWs attn_dec_layout(const AttnShape& a) {
  AttnDecWs w;
  w.chunk = attn_decode_chunk(a.D, a.B, a.Hkv, (a.H / a.Hkv + kAttnDecHeads - 1) / kAttnDecHeads, std::max(a.S, 1));
  w.nchunks = (std::max(a.S, 1) + w.chunk - 1) / w.chunk;
  const size_t slots = static_cast<size_t>(a.B) * a.H * w.nchunks;
  w.part_o = 0;
  w.part_ml = align_up(sizeof(float) * slots * a.D);
  w.end = align_up(w.part_ml + sizeof(float) * 2 * slots);
  return w;
}
}  // namespace
}  // extern "C++"

star_status star_attn_fwd(const star_attn_shape* shape, const void* plan, const void* Q, const void* K,
                          const void* V, star_dtype dt, void* O, star_dtype ot, float* lse, hipStream_t stream) {
  AttnShape a;
  star_status st = parse_attn(shape, a);
  if (st != STAR_OK) return st;
  if (dt != STAR_BF16 || !valid_dtype(ot)) return STAR_ERR_DTYPE;
  if (a.B == 0 || a.S == 0) return STAR_OK;
  if (!plan || !Q || !K || !V || !O) return STAR_ERR_ARG;
  if (!aligned16(plan) || !aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(O)) return STAR_ERR_ALIGN;
  if (lse && !aligned4(lse)) return STAR_ERR_ALIGN;
  if (a.S > kAttnFwdMaxSeq) return STAR_ERR_SHAPE;
  const int64_t items = attn_fwd_items(a.S, a.q);
  if (static_cast<int64_t>(a.B) * a.H * items > 0x7fffffff) return STAR_ERR_SHAPE;
  const PlanWs pw = plan_layout(a.S, a.q);
  AttnParams p = attn_params(a);
  p.Q = Q;
  p.K = K;
  p.V = V;
  p.O = O;
  p.odtype = ot == STAR_BF16 ? 1 : 0;
  p.lse = lse;
  p.perm = at<int32_t>(const_cast<void*>(plan), pw.perm);
  p.offsets = at<int32_t>(const_cast<void*>(plan), pw.offsets);
  p.items_per_bh = static_cast<int32_t>(items);
  return hip_status(launch_attn_fwd(p, stream));
}

size_t star_attn_decode_workspace_bytes(const star_attn_shape* shape) {
  AttnShape a;
  if (parse_attn(shape, a) != STAR_OK) return 0;
  return attn_dec_layout(a).end;
}

star_status star_attn_decode(const star_attn_shape* shape, const int32_t* pos_type, const int32_t* cache_len,
                             const void* Q, const void* K_cache, const void* V_cache, star_dtype dt, void* O,
                             star_dtype ot, void* ws, size_t ws_bytes, hipStream_t stream) {
  AttnShape a;
  star_status st = parse_attn(shape, a);
  if (st != STAR_OK) return st;
  if (dt != STAR_BF16 || !valid_dtype(ot)) return STAR_ERR_DTYPE;
  if (a.B == 0) return STAR_OK;
  if (a.S == 0) return STAR_ERR_SHAPE;  // a decode step needs a cache
  if (!pos_type || !cache_len || !Q || !K_cache || !V_cache || !O) return STAR_ERR_ARG;
  if (!aligned4(pos_type) || !aligned4(cache_len)) return STAR_ERR_ALIGN;
  if (!aligned16(Q) || !aligned16(K_cache) || !aligned16(V_cache) || !aligned16(O)) return STAR_ERR_ALIGN;
  const AttnDecWs w = attn_dec_layout(a);
  if (!ws || ws_bytes < w.end) return STAR_ERR_WORKSPACE;
  if (!aligned16(ws)) return STAR_ERR_ALIGN;
  AttnParams p = attn_params(a);
  p.head_groups = (a.H / a.Hkv + kAttnDecHeads - 1) / kAttnDecHeads;
  if (a.B > 65535 || w.nchunks > 65535) return STAR_ERR_SHAPE;
  p.Q = Q;
  p.K = K_cache;
  p.V = V_cache;
  p.O = O;
  p.odtype = ot == STAR_BF16 ? 1 : 0;
  p.pos_type = pos_type;
  p.cache_len = cache_len;
  p.chunk = w.chunk;
  p.nchunks = w.nchunks;
  p.part_o = at<float>(ws, w.part_o);
  p.part_ml = at<float>(ws, w.part_ml);
  return hip_status(launch_attn_decode(p, stream));
}

}  // extern "C"
