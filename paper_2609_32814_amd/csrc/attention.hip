// Algebraic attention (appendix "Attention Extension and Detailed Cost
// Accounting"): causal attention whose query-key score keeps only the feature
// groups F(i, j) of the two positions' types (eq. feature-set; eq.
// tensor-square-feature-set for the tensor power), scaled by 1 / sqrt(|F| m)
// (eqs. attention-support-size, attention-score), with the causal mask and
// dense value aggregation (eqs. causal-mask, softmax-pv).
//
// Forward (Alg. attention-training, the score and aggregation steps).  The
// positions of a sequence are grouped by type through the stable type plan of
// the position-type table (the same for every sequence).  A workgroup of 4
// wavefronts owns one block of up to 128 query positions of one type i of
// one (sequence, head), 32 per wave, and walks the keys type by type in
// blocks of 32.  Positions increase within a type, so the first key block
// that starts past the workgroup's last query ends that type's walk.  Per key
// block of type j:
//   S^T = K Q^T over the groups of F(i, j) only, with
//         v_mfma_f32_32x32x16_bf16: the key rows are the A operand (read from
//         global memory, 16 bytes a lane), the wave's query rows the B
//         operand (held in registers for the whole walk), so a lane ends with
//         16 key scores of one query.  Contraction steps whose 16 features
//         hold no selected group are skipped; with m = 8 a lane zeroes its
//         own 8-feature slice when that group is not selected;
//   base-2 scaling, the causal mask, and the online softmax (row max and
//         sum over the lane's 16 values and its partner lane l ^ 32, which
//         holds the other 16 keys of the same query);
//   O^T += V^T P^T: the probabilities stay in registers as the B operand;
//         the value block reaches LDS by direct global-to-LDS copies (issued
//         before the score step, so they overlap it) and is read back with
//         transposing reads (ds_read_b64_tr_b16) in exactly the key order in
//         which the lane holds its probabilities.
//
// Decode (Alg. attention-decoding, the score and aggregation steps) splits
// the cache into chunks: a workgroup takes one chunk of one sequence for one
// key/value head and up to 8 of its query heads, so each cached key and
// value row is read once for all of them.  Teams of head_dim / 8 lanes take a
// key each (16 bytes a lane): a lane whose 8 features belong to no selected
// group of that key reads nothing.  Scores go to LDS, the chunk's softmax
// runs there, the value rows are weighted in registers and the teams are
// summed in LDS in a fixed order.  A second kernel merges the chunks of a
// (sequence, head) by their maxima and sums.
#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"

namespace starq {

namespace {

typedef short v4i16_t __attribute__((ext_vector_type(4)));
#define STARQ_LDS __attribute__((address_space(3)))

constexpr int kQRows = 32;        // query rows per MFMA tile
constexpr int kBlockRows = 128;   // query rows per workgroup

__device__ __attribute__((aligned(256))) uint32_t g_attn_zero[64];

__device__ __forceinline__ void dma16(const void* g, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" : : "v"(g), "s"(lds_addr) : "memory", "m0");
}
__device__ __forceinline__ void wait_vm_all() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));  // vmcnt(0)
  asm volatile("" ::: "memory");
}
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(reinterpret_cast<uintptr_t>(p)));
}

// a in F(i, j): star (law 0) {i, j}; dense (law 1) every group; tensor power
// (law 2) every bit of a equal to that bit of i or of j.
__device__ __forceinline__ bool attn_in_group(int law, int i, int j, int a) {
  if (law == 1) return true;
  if (law == 2) return ((a ^ i) & (a ^ j)) == 0;
  return a == i || a == j;
}
__device__ __forceinline__ uint32_t attn_fmask(int law, int q, int i, int j) {
  uint32_t f = 0;
  for (int a = 0; a < q; ++a)
    if (attn_in_group(law, i, j, a)) f |= 1u << a;
  return f;
}

typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// Two fp32 values rounded to bf16 (nearest even) and packed, low half first:
// one v_cvt_pk_bf16_f32.
// max / sum of a value and its partner lane l ^ 32 (v_permlane32_swap; both
// lanes get the same result)
__device__ __forceinline__ float max_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a, b}, bf16x2_t));
}

// LDS tiles of one 64-key step: a plane per 16-byte feature chunk, each
// plane the chunk of the 64 key rows in row order (1 KB, exactly one
// global-to-LDS copy with lane = row), padded to kPlane bytes so that the
// transposing reads of neighbouring planes fall on different banks.  The key
// tile holds only the chunks of the selected groups F(i, j), packed in
// chunk order; the value tile holds every chunk.
constexpr int kStepKeys = 64;
// 64-key blocks over all types the forward can index (positions up to
// kAttnFwdMaxSeq plus a partial block per type), rounded up to the 256 block
// flags one pass of a 256-thread workgroup writes
constexpr int kFwdMaxBlocks = (kAttnFwdMaxSeq / kStepKeys + 32 + 255) / 256 * 256;
constexpr int kPlane = 1024 + 64;

template <int DH>
constexpr int fwd_tile_bytes() { return (DH / 8) * kPlane; }
template <int DH>
constexpr int fwd_smem() { return 2 * 2 * fwd_tile_bytes<DH>(); }  // two stages of (K, V)

// Query tiles of 32 rows per wave (one: four waves per 128-row block).
template <int DH>
constexpr int fwd_qtiles() { return 1; }
template <int DH>
constexpr int fwd_threads() { return 64 * (kBlockRows / (kQRows * fwd_qtiles<DH>())); }

// M8: groups of 8 features (two groups per 16-feature contraction step).
template <int DH, bool M8>
__global__ __launch_bounds__(fwd_threads<DH>()) void attn_fwd_kernel(const AttnParams p) {
  constexpr int QT = fwd_qtiles<DH>();    // 32-row query tiles per wave
  constexpr int NW = fwd_threads<DH>() / 64;
  constexpr int NT = NW * 64;
  constexpr int NCH = DH / 32;  // 32-feature output chunks
  constexpr int KS = DH / 16;   // 16-feature contraction steps over a head
  constexpr int CPR = DH / 8;   // 16-byte chunks (planes) per row
  constexpr int TILE = fwd_tile_bytes<DH>();
  extern __shared__ __attribute__((aligned(16))) char tiles[];  // [stage][K, V][planes]
  __shared__ int32_t qpos_s[kBlockRows];
  __shared__ int32_t kpos_s[2][kStepKeys];
  __shared__ int32_t off_s[32 + 1];
  __shared__ int32_t nstep_s[32];
  __shared__ uint64_t bits_s[kFwdMaxBlocks / 64];
  // per key type j: F(i, j) as a group mask, the selected chunks as a mask,
  // their count, the score scale (bits), then the selected chunks in order
  __shared__ uint32_t tab_s[32][4 + 16];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lr = lane & 31, lh = lane >> 5;
  const int q = p.q, m = DH / q, cpg = m / 8;

  // ---- work item.  Workgroup w runs on XCD w % 8 (round-robin dispatch);
  // each XCD takes a contiguous range of (sequence, head) pairs, so the query
  // blocks of one pair run side by side and share its keys and values in that
  // XCD's L2.  Within a pair the latest (longest) query blocks come first.
  const int32_t BH = p.B * p.n_heads;
  const int64_t n_items = static_cast<int64_t>(BH) * p.items_per_bh;
  const int64_t per_xcd = (n_items + 7) / 8;
  const int64_t item = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
  if (item >= n_items) return;
  const int32_t bh = static_cast<int32_t>(item / p.items_per_bh);
  int32_t r = static_cast<int32_t>(item % p.items_per_bh);
  int i = -1;
  int32_t qb = 0;
  for (int32_t lvl = 0; i < 0; ++lvl) {
    bool any = false;
    for (int t = 0; t < q; ++t) {
      const int32_t nbt = (p.offsets[t + 1] - p.offsets[t] + kBlockRows - 1) / kBlockRows;
      if (nbt > lvl) {
        any = true;
        if (r == 0) {
          i = t;
          qb = nbt - 1 - lvl;
          break;
        }
        --r;
      }
    }
    if (!any) break;
  }
  if (i < 0) return;  // past the last block (uniform over the workgroup)
  const int b = bh / p.n_heads, h = bh % p.n_heads;
  const int32_t q0 = p.offsets[i] + qb * kBlockRows;
  const int32_t qend = p.offsets[i + 1];
  const int hk = h / (p.n_heads / p.n_kv);
  const int64_t ldq = static_cast<int64_t>(p.n_heads) * DH, ldk = static_cast<int64_t>(p.n_kv) * DH;
  const uint16_t* Qg = static_cast<const uint16_t*>(p.Q) + static_cast<int64_t>(b) * p.S * ldq + h * DH;
  const uint16_t* Kg = static_cast<const uint16_t*>(p.K) + static_cast<int64_t>(b) * p.S * ldk + hk * DH;
  const uint16_t* Vg = static_cast<const uint16_t*>(p.V) + static_cast<int64_t>(b) * p.S * ldk + hk * DH;

  // ---- prologue: one round of global loads (the block's query positions,
  // its last query, the first position of every 64-key block of every type,
  // and the key rows of the first two blocks of type 0, the likely first
  // steps), then the step counts.
  const int32_t nvalid = min(kBlockRows, qend - q0);
  const int32_t wg_last = p.perm[q0 + nvalid - 1];
  for (int x = threadIdx.x; x < kBlockRows; x += NT) {
    const int32_t pos = q0 + x;
    qpos_s[x] = pos < qend ? p.perm[pos] : -1;
  }
  if (threadIdx.x <= q) off_s[threadIdx.x] = p.offsets[threadIdx.x];
  // Groups are taken in the rotated order a' = (a - i) mod q, so that the
  // query's own group i, which every F(i, j) holds, comes first: the first
  // contraction step of every key tile is then always selected.
  if (threadIdx.x < q) {
    const int j = threadIdx.x;
    const uint32_t fm = attn_fmask(p.law, q, i, j);
    uint32_t csel = 0;  // selected chunks, rotated order
    int n = 0;
    for (int ar = 0; ar < q; ++ar) {
      const int a = (ar + i) % q;
      if ((fm >> a) & 1u) {
        csel |= ((1u << cpg) - 1u) << (ar * cpg);
        for (int c = 0; c < cpg; ++c) tab_s[j][4 + n++] = a * cpg + c;
      }
    }
    tab_s[j][0] = fm;
    tab_s[j][1] = csel;
    tab_s[j][2] = n;
    tab_s[j][3] = __float_as_uint(kLog2e * __builtin_amdgcn_rsqf(static_cast<float>(__popc(fm) * m)));
  }
  const int32_t off0 = p.offsets[0], off1 = p.offsets[1];
  int32_t kp_cur = off0 + lane < off1 ? p.perm[off0 + lane] : 0x7fffffff;
  int32_t kp_nxt = off0 + kStepKeys + lane < off1 ? p.perm[off0 + kStepKeys + lane] : 0x7fffffff;
  // one bit per 64-key block, all types in order: does the block start at
  // or before the workgroup's last query?
  int32_t NB = 0;
  for (int j = 0; j < q; ++j) NB += (p.offsets[j + 1] - p.offsets[j] + kStepKeys - 1) / kStepKeys;
  for (int32_t x0 = 0; x0 < NB; x0 += NT) {
    const int32_t x = x0 + threadIdx.x;
    int32_t first = 0x7fffffff;
    int32_t base = 0;
    for (int j = 0; j < q; ++j) {
      const int32_t oj = p.offsets[j], nb = (p.offsets[j + 1] - oj + kStepKeys - 1) / kStepKeys;
      if (x >= base && x < base + nb) first = p.perm[oj + kStepKeys * (x - base)];
      base += nb;
    }
    const uint64_t bal = __ballot(first <= wg_last);
    if (lane == 0) bits_s[(x0 >> 6) + wave] = bal;
  }
  __syncthreads();
  // steps of type j: the set bits among its blocks
  if (threadIdx.x < q) {
    const int j = threadIdx.x;
    int32_t base = 0;
    for (int t = 0; t < j; ++t) base += (off_s[t + 1] - off_s[t] + kStepKeys - 1) / kStepKeys;
    const int32_t nb = (off_s[j + 1] - off_s[j] + kStepKeys - 1) / kStepKeys;
    int32_t n = 0;
    for (int32_t x = base; x < base + nb;) {
      const int32_t w = x >> 6, lo = x & 63, hi = min(64, lo + (base + nb - x));
      uint64_t word = bits_s[w] >> lo;
      if (hi - lo < 64) word &= (1ull << (hi - lo)) - 1ull;
      n += __popcll(word);
      x += hi - lo;
    }
    nstep_s[j] = n;
  }
  // positions increase along the block: the first and last query of each of
  // the wave's tiles (read through readfirstlane: the compiler then branches
  // on them as wave-uniform values)
  int32_t tfirst[QT], tlast[QT], my_qpos[QT];
#pragma unroll
  for (int u = 0; u < QT; ++u) {
    const int row0 = (wave * QT + u) * kQRows;
    const int32_t tv = min(kQRows, nvalid - row0);  // valid rows of this tile (may be <= 0)
    tfirst[u] = tv > 0 ? __builtin_amdgcn_readfirstlane(qpos_s[row0]) : 0x7fffffff;
    tlast[u] = tv > 0 ? __builtin_amdgcn_readfirstlane(qpos_s[row0 + tv - 1]) : -1;
    my_qpos[u] = qpos_s[row0 + lr];
  }
  const int32_t wave_last = tlast[QT - 1] >= 0 ? tlast[QT - 1] : tlast[0];

  // the wave's query rows as B operands: for rotated step ks lane half lh
  // holds the 8 features at rotated position 16 ks + 8 lh of row lr of each
  // tile, i.e. offset o of rotated group a' (physical group (a' + i) mod q)
  uint4 qf[QT][KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    const int fr = 16 * ks + 8 * lh;
    const int fphys = ((fr / m + i) % q) * m + fr % m;
#pragma unroll
    for (int u = 0; u < QT; ++u) {
      qf[u][ks] = make_uint4(0, 0, 0, 0);
      if (my_qpos[u] >= 0) qf[u][ks] = *reinterpret_cast<const uint4*>(Qg + static_cast<int64_t>(my_qpos[u]) * ldq + fphys);
    }
  }
  __syncthreads();
  // step counts and offsets are the same for every lane: readfirstlane makes
  // the step loop and its branches scalar
  auto nsteps = [&](int j) { return __builtin_amdgcn_readfirstlane(nstep_s[j]); };
  auto tab = [&](int j, int f) { return static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(tab_s[j][f])); };
  auto offs = [&](int j) { return __builtin_amdgcn_readfirstlane(off_s[j]); };
  int32_t T = 0;
  for (int j = 0; j < q; ++j) T += nsteps(j);

  // step iterator: (type, block), skipping types without steps
  struct It {
    int j;
    int32_t c;
  };
  auto normalize = [&](It& it) {
    while (it.j < q && it.c >= nsteps(it.j)) {
      ++it.j;
      it.c = 0;
    }
  };
  auto advance = [&](It& it) {
    ++it.c;
    normalize(it);
  };
  // the position of this lane's key row in a step (INT_MAX past the type's end)
  auto load_kp = [&](const It& it) -> int32_t {
    if (it.j >= q) return 0x7fffffff;
    const int32_t k = offs(it.j) + kStepKeys * it.c + lane;
    return k < offs(it.j + 1) ? p.perm[k] : 0x7fffffff;
  };
  // global-to-LDS copies of a step's key planes (selected chunks only) and
  // value planes; lane = key row
  const void* zero = g_attn_zero;
  auto issue = [&](const It& it, int32_t kp, int stage) {
    char* Kt = tiles + stage * 2 * TILE;
    char* Vt = Kt + TILE;
    const int nsel = static_cast<int>(tab(it.j, 2));
    const bool ok = kp < p.S;
    const uint16_t* krow = Kg + static_cast<int64_t>(ok ? kp : 0) * ldk;
    const uint16_t* vrow = Vg + static_cast<int64_t>(ok ? kp : 0) * ldk;
    for (int k = wave; k < nsel; k += NW) {
      const int c = static_cast<int>(tab(it.j, 4 + k));
      dma16(ok ? static_cast<const void*>(krow + 8 * c) : zero, lds_addr(Kt + k * kPlane));
    }
    for (int c = wave; c < CPR; c += NW)
      dma16(ok ? static_cast<const void*>(vrow + 8 * c) : zero, lds_addr(Vt + c * kPlane));
  };

  // online softmax state of the lane's query in each tile (shared with lane
  // l ^ 32)
  float run_max[QT], run_sum[QT];
  f32x16_t acc[QT][NCH];
#pragma unroll
  for (int u = 0; u < QT; ++u) {
    run_max[u] = -INFINITY;
    run_sum[u] = 0.f;
#pragma unroll
    for (int c = 0; c < NCH; ++c)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[u][c][e] = 0.f;
  }

  It cur{0, 0};
  normalize(cur);
  It nxt = cur;
  advance(nxt);
  // the speculative rows were those of type 0, blocks 0 and 1
  if (cur.j != 0 || cur.c != 0) kp_cur = load_kp(cur);
  if (nxt.j != 0 || nxt.c != 1) kp_nxt = load_kp(nxt);
  if (T > 0) {
    wait_vm_all();
    if (wave == 0) kpos_s[0][lane] = kp_cur;
    issue(cur, kp_cur, 0);
  }
  for (int32_t s = 0; s < T; ++s) {
    wait_vm_all();    // this step's copies and the next step's positions
    __syncthreads();  // the tiles of step s are visible; step s - 1 is done everywhere
    It nn = nxt;
    advance(nn);
    if (s + 1 < T) {
      if (wave == 0) kpos_s[(s + 1) & 1][lane] = kp_nxt;
      issue(nxt, kp_nxt, (s + 1) & 1);
      kp_nxt = load_kp(nn);
    }

    const char* Kt = tiles + (s & 1) * 2 * TILE;
    const char* Vt = Kt + TILE;
    const int32_t* kps = kpos_s[s & 1];
    // chunk c of the head is plane popc(csel below c) of the key tile
    const uint32_t csel = tab(cur.j, 1);
    const float scale = __uint_as_float(tab(cur.j, 3));
    // first and last keys of the two halves (uniform)
    const int32_t kf0 = __builtin_amdgcn_readfirstlane(kps[0]), kf1 = __builtin_amdgcn_readfirstlane(kps[32]);
    const int32_t kl0 = __builtin_amdgcn_readfirstlane(kps[31]), kl1 = __builtin_amdgcn_readfirstlane(kps[63]);
    if (kf0 <= wave_last) {  // some key of the step precedes a query of the wave
      // Every query tile and both key halves are computed; keys after a
      // query are removed by the causal mask (a half past the type's end has
      // positions INT_MAX).
      f32x16_t sc[QT][2];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const char* Krow = Kt + (32 * t + lr) * 16;
        // rotated step ks uses key planes popc(csel below 2 ks) + lh; step 0
        // (the query's own group) is always selected and starts the sum
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          if (ks > 0 && !((csel >> (2 * ks)) & 3u)) continue;
          uint4 kf;
          if constexpr (!M8) {
            // m >= 16: a step's 16 features lie in one group
            const int pl = __popc(csel & ((1u << (2 * ks)) - 1u)) + lh;
            kf = *reinterpret_cast<const uint4*>(Krow + pl * kPlane);
          } else {
            // m = 8: the halves of a step are two groups; a lane whose group
            // is not selected reads plane 0 and contributes zeros
            const int c = 2 * ks + lh;
            const bool on = (csel >> c) & 1u;
            const int pl = on ? __popc(csel & ((1u << c) - 1u)) : 0;
            kf = *reinterpret_cast<const uint4*>(Krow + pl * kPlane);
            if (!on) kf = make_uint4(0, 0, 0, 0);
          }
#pragma unroll
          for (int u = 0; u < QT; ++u) {
            if (ks == 0)
              sc[u][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, kf),
                                                                 __builtin_bit_cast(bf16x8_t, qf[u][0]), f32x16_t{}, 0, 0, 0);
            else
              sc[u][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, kf),
                                                                 __builtin_bit_cast(bf16x8_t, qf[u][ks]), sc[u][t], 0, 0, 0);
          }
        }
      }
      // lane holds query lr of tile u against keys 32 t + 8 (e / 4) + 4 lh + e % 4
      bool need_any = false;
      float bmax[QT];
#pragma unroll
      for (int u = 0; u < QT; ++u) {
        bmax[u] = -INFINITY;
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          // the causal mask is needed only where a key of this half follows
          // the tile's first query
          if ((t ? kl1 : kl0) > tfirst[u]) {
#pragma unroll
            for (int a = 0; a < 4; ++a) {
              const int4 kq = *reinterpret_cast<const int4*>(kps + 32 * t + 8 * a + 4 * lh);
              if (kq.x > my_qpos[u]) sc[u][t][4 * a + 0] = -INFINITY;
              if (kq.y > my_qpos[u]) sc[u][t][4 * a + 1] = -INFINITY;
              if (kq.z > my_qpos[u]) sc[u][t][4 * a + 2] = -INFINITY;
              if (kq.w > my_qpos[u]) sc[u][t][4 * a + 3] = -INFINITY;
            }
          }
#pragma unroll
          for (int e = 0; e < 16; ++e) bmax[u] = fmaxf(bmax[u], sc[u][t][e]);
        }
        // the step's largest scaled score (base 2) of the lane's query
        bmax[u] = max_xor32(bmax[u]) * scale;
        need_any |= bmax[u] > run_max[u] + 8.f;
      }
      // Lazy rescaling: the running maximum moves (and the accumulators are
      // rescaled) only when a score exceeds it by more than 8, so every
      // probability stays below 2^8; the normalisation by the sum at the end
      // is unchanged.  A row whose keys so far are all masked keeps -inf.
      if (__ballot(need_any) != 0) {
#pragma unroll
        for (int u = 0; u < QT; ++u) {
          const bool need = bmax[u] > run_max[u] + 8.f;
          const float corr = need ? __builtin_amdgcn_exp2f(run_max[u] - bmax[u]) : 1.f;
          if (need) run_max[u] = bmax[u];
          run_sum[u] *= corr;
#pragma unroll
          for (int c = 0; c < NCH; ++c)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[u][c][e] *= corr;
        }
      }
      // probabilities, packed to bf16 as the B operands of the value product:
      // pf[u][kk] holds the keys 16 kk + 4 lh + 0..3 and 16 kk + 8 + 4 lh + 0..3
      uint4 pf[QT][4];
#pragma unroll
      for (int u = 0; u < QT; ++u) {
        const float base = run_max[u] == -INFINITY ? 0.f : run_max[u];
        float bsum = 0.f;
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          float pe[16];
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            pe[e] = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[u][t][e], scale, -base));
            bsum += pe[e];
          }
#pragma unroll
          for (int k2 = 0; k2 < 2; ++k2)
            pf[u][2 * t + k2] = make_uint4(pack_bf16(pe[8 * k2 + 0], pe[8 * k2 + 1]), pack_bf16(pe[8 * k2 + 2], pe[8 * k2 + 3]),
                                           pack_bf16(pe[8 * k2 + 4], pe[8 * k2 + 5]), pack_bf16(pe[8 * k2 + 6], pe[8 * k2 + 7]));
        }
        run_sum[u] += sum_xor32(bsum);
      }

      // O^T += V^T P^T in 16-key steps; each value fragment serves every
      // query tile
      const int g = lane >> 4, pp = lane & 15;
      const int rr = pp >> 2, qq = pp & 3;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const int row0 = 16 * kk + 4 * (g >> 1) + rr;
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
          // in 16-lane group g, lanes 4 rr + qq address features f .. f + 3
          // of key rows row0 and row0 + 8; lane pp receives feature
          // 32 c + 16 (g & 1) + pp of those 4 + 4 rows
          const int f = 32 * c + 16 * (g & 1) + 4 * qq;
          const char* a0 = Vt + (f >> 3) * kPlane + row0 * 16 + ((f >> 2) & 1) * 8;
          const uint2 w0 = __builtin_bit_cast(uint2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((STARQ_LDS v4i16_t*)(a0)));
          const uint2 w1 = __builtin_bit_cast(uint2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((STARQ_LDS v4i16_t*)(a0 + 8 * 16)));
          const uint4 vf = make_uint4(w0.x, w0.y, w1.x, w1.y);
#pragma unroll
          for (int u = 0; u < QT; ++u)
              acc[u][c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, vf),
                                                                  __builtin_bit_cast(bf16x8_t, pf[u][kk]), acc[u][c], 0, 0, 0);
        }
      }
    }
    cur = nxt;
    nxt = nn;
  }

  // ---- O = acc / sum: lane holds query lr of each tile, features
  // 32 c + 8 a + 4 lh + 0..3
#pragma unroll
  for (int u = 0; u < QT; ++u) {
    if (my_qpos[u] < 0) continue;
    const float inv = run_sum[u] > 0.f ? 1.f / run_sum[u] : 0.f;
    const int64_t o = (static_cast<int64_t>(b) * p.S + my_qpos[u]) * ldq + h * DH;
#pragma unroll
    for (int c = 0; c < NCH; ++c)
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        const int f = 32 * c + 8 * a + 4 * lh;
        const float v0 = acc[u][c][4 * a] * inv, v1 = acc[u][c][4 * a + 1] * inv;
        const float v2 = acc[u][c][4 * a + 2] * inv, v3 = acc[u][c][4 * a + 3] * inv;
        if (p.odtype == 0) {
          *reinterpret_cast<float4*>(static_cast<float*>(p.O) + o + f) = make_float4(v0, v1, v2, v3);
        } else {
          *reinterpret_cast<uint2*>(static_cast<uint16_t*>(p.O) + o + f) = make_uint2(pack_bf16(v0, v1), pack_bf16(v2, v3));
        }
      }
    if (p.lse && lh == 0) {
      const float l = run_sum[u] > 0.f ? (run_max[u] + __log2f(run_sum[u])) * 0.6931471805599453f : -INFINITY;
      p.lse[(static_cast<int64_t>(b) * p.n_heads + h) * p.S + my_qpos[u]] = l;
    }
  }
}

// ---- decode ---------------------------------------------------------------------

constexpr int kDecThreads = 256;
constexpr int kDecBatch = 4;  // keys per team per batch (loads issued together)
constexpr int kDecMaxChunk = 8 * kDecBatch * kDecThreads / 8;  // the longest chunk (head width 64)

// One chunk of the cache of one sequence against up to G query heads that
// share one key/value head.  Teams of T = DH / 8 lanes take the keys
// u0 + team + NT k in order, a batch of 4 at a time, and keep an online
// softmax per head in registers (running base-2 maximum, sum, and the lane's
// 8 output features); the teams are merged at the end through LDS.
template <int DH, int G>
__global__ __launch_bounds__(kDecThreads) void attn_decode_part_kernel(const AttnParams p) {
  constexpr int T = DH / 8;            // lanes per key
  constexpr int NT = kDecThreads / T;  // teams
  extern __shared__ __attribute__((aligned(16))) float dsm[];  // [NT][gh][DH + 2] team states
  __shared__ uint32_t fm_s[32];        // F(i, j) as a bit mask, per key type j
  __shared__ int32_t types_s[kDecMaxChunk];  // types of the chunk's positions

  // the head index varies fastest over the grid: workgroups dispatched
  // together read the same cache rows (all heads of a position are adjacent)
  const int chunk = blockIdx.y;
  const int hk = blockIdx.x / p.head_groups, hg = blockIdx.x % p.head_groups;
  const int b = blockIdx.z;
  const int g_all = p.n_heads / p.n_kv;
  const int h0 = hk * g_all + hg * kAttnDecHeads;
  const int gh = min(G, g_all - hg * kAttnDecHeads);
  const int q = p.q, m = DH / q;
  const int32_t L = min(p.cache_len[b], p.S);
  const int32_t u0 = chunk * p.chunk;
  if (L <= 0 || u0 >= L) return;
  const int i = p.pos_type[L - 1];
  if (static_cast<unsigned>(i) >= static_cast<unsigned>(q)) return;  // the merge writes zeros
  const int32_t u1 = min(L, u0 + p.chunk);
  const int tid = threadIdx.x;
  const int team = tid / T, t = tid % T;
  if (tid < q) fm_s[tid] = attn_fmask(p.law, q, i, tid);
  for (int32_t r = tid; r < u1 - u0; r += kDecThreads) types_s[r] = p.pos_type[u0 + r];

  const int64_t ldq = static_cast<int64_t>(p.n_heads) * DH, ldk = static_cast<int64_t>(p.n_kv) * DH;
  const uint16_t* Kc = static_cast<const uint16_t*>(p.K) + static_cast<int64_t>(b) * p.S * ldk + hk * DH + 8 * t;
  const uint16_t* Vc = static_cast<const uint16_t*>(p.V) + static_cast<int64_t>(b) * p.S * ldk + hk * DH + 8 * t;
  // the lane's 8 query features of each head
  float qf[G][8];
#pragma unroll
  for (int hh = 0; hh < G; ++hh) {
    uint4 v = make_uint4(0, 0, 0, 0);
    if (hh < gh) v = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(p.Q) + b * ldq + (h0 + hh) * DH + 8 * t);
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      qf[hh][2 * e] = bf16_to_f32(w[e] & 0xffffu);
      qf[hh][2 * e + 1] = bf16_to_f32(w[e] >> 16);
    }
  }
  __syncthreads();
  const int al = (8 * t) / m;  // the lane's feature group

  float mrun[G], lrun[G], o[G][8];
#pragma unroll
  for (int hh = 0; hh < G; ++hh) {
    mrun[hh] = -INFINITY;
    lrun[hh] = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) o[hh][e] = 0.f;
  }
  // key u of batch kb of this team: ub(kb) + NT k with ub(kb) = u0 + team +
  // kBatch NT kb; its type (or -1 past the chunk) from LDS
  const int32_t n = u1 - u0;
  const int nb = (n - team + kDecBatch * NT - 1) / (kDecBatch * NT);  // batches of this team
  struct Batch {
    uint4 kv[kDecBatch], vv[kDecBatch];
    int32_t jt[kDecBatch];
  };
  auto load = [&](int kb, Batch& bt) {
#pragma unroll
    for (int k = 0; k < kDecBatch; ++k) {
      const int32_t r = team + NT * (kDecBatch * kb + k);  // position within the chunk
      const int32_t j = r < n ? types_s[r] : -1;
      bt.jt[k] = j;
      const bool key_ok = static_cast<unsigned>(j) < static_cast<unsigned>(q);
      const int64_t u = u0 + r;
      bt.kv[k] = make_uint4(0, 0, 0, 0);
      bt.vv[k] = make_uint4(0, 0, 0, 0);
      if (key_ok && ((fm_s[key_ok ? j : 0] >> al) & 1u)) bt.kv[k] = *reinterpret_cast<const uint4*>(Kc + u * ldk);
      if (key_ok) bt.vv[k] = *reinterpret_cast<const uint4*>(Vc + u * ldk);
    }
  };
  auto compute = [&](const Batch& bt) {
    // scores (base 2), -inf for keys past the chunk or of an out-of-range type
    float sc[kDecBatch][G];
#pragma unroll
    for (int k = 0; k < kDecBatch; ++k) {
      const uint32_t w[4] = {bt.kv[k].x, bt.kv[k].y, bt.kv[k].z, bt.kv[k].w};
      float kf[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        kf[2 * e] = bf16_to_f32(w[e] & 0xffffu);
        kf[2 * e + 1] = bf16_to_f32(w[e] >> 16);
      }
#pragma unroll
      for (int hh = 0; hh < G; ++hh) {
        float a = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) a += qf[hh][e] * kf[e];
        sc[k][hh] = a;
      }
#pragma unroll
      for (int o2 = T / 2; o2 > 0; o2 >>= 1)
#pragma unroll
        for (int hh = 0; hh < G; ++hh) sc[k][hh] += __shfl_xor(sc[k][hh], o2, T);
      const bool key_ok = static_cast<unsigned>(bt.jt[k]) < static_cast<unsigned>(q);
      const float scale = key_ok ? kLog2e * __builtin_amdgcn_rsqf(static_cast<float>(__popc(fm_s[key_ok ? bt.jt[k] : 0]) * m)) : 0.f;
#pragma unroll
      for (int hh = 0; hh < G; ++hh) sc[k][hh] = key_ok ? sc[k][hh] * scale : -INFINITY;
    }
    // online softmax update per head
#pragma unroll
    for (int hh = 0; hh < G; ++hh) {
      float bm = sc[0][hh];
#pragma unroll
      for (int k = 1; k < kDecBatch; ++k) bm = fmaxf(bm, sc[k][hh]);
      const float nm = fmaxf(mrun[hh], bm);
      if (nm == -INFINITY) continue;  // nothing valid yet (team-uniform)
      const float corr = __builtin_amdgcn_exp2f(mrun[hh] - nm);
      mrun[hh] = nm;
      lrun[hh] *= corr;
#pragma unroll
      for (int e = 0; e < 8; ++e) o[hh][e] *= corr;
#pragma unroll
      for (int k = 0; k < kDecBatch; ++k) {
        const float pk = __builtin_amdgcn_exp2f(sc[k][hh] - nm);
        lrun[hh] += pk;
        const uint32_t w[4] = {bt.vv[k].x, bt.vv[k].y, bt.vv[k].z, bt.vv[k].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          o[hh][2 * e] += pk * bf16_to_f32(w[e] & 0xffffu);
          o[hh][2 * e + 1] += pk * bf16_to_f32(w[e] >> 16);
        }
      }
    }
  };
  // two batches in flight: the next batch's rows are requested before the
  // current one is used
  Batch b0, b1;
  if (nb > 0) load(0, b0);
  for (int kb = 0; kb < nb; kb += 2) {
    if (kb + 1 < nb) load(kb + 1, b1);
    compute(b0);
    if (kb + 1 >= nb) break;
    if (kb + 2 < nb) load(kb + 2, b0);
    compute(b1);
  }
  // ---- merge the teams: state of team tm, head hh at dsm[(tm gh + hh)(DH + 2)]
#pragma unroll
  for (int hh = 0; hh < G; ++hh) {
    if (hh >= gh) break;
    float* dst = dsm + (static_cast<int64_t>(team) * gh + hh) * (DH + 2);
#pragma unroll
    for (int e = 0; e < 8; ++e) dst[8 * t + e] = o[hh][e];
    if (t == 0) {
      dst[DH] = mrun[hh];
      dst[DH + 1] = lrun[hh];
    }
  }
  __syncthreads();
  const int64_t slot0 = (static_cast<int64_t>(b) * p.n_heads + h0) * p.nchunks + chunk;
  for (int x = tid; x < gh * DH; x += kDecThreads) {
    const int hh = x / DH, f = x % DH;
    float M = -INFINITY;
    for (int tm = 0; tm < NT; ++tm) M = fmaxf(M, dsm[(tm * gh + hh) * (DH + 2) + DH]);
    float a = 0.f, l = 0.f;
    if (M != -INFINITY)
      for (int tm = 0; tm < NT; ++tm) {
        const float* st = dsm + (tm * gh + hh) * (DH + 2);
        const float w = __builtin_amdgcn_exp2f(st[DH] - M);
        a += w * st[f];
        l += w * st[DH + 1];
      }
    const int64_t sl = slot0 + static_cast<int64_t>(hh) * p.nchunks;
    p.part_o[sl * DH + f] = a;
    if (f == 0) {
      p.part_ml[2 * sl] = M;
      p.part_ml[2 * sl + 1] = l;
    }
  }
}

// Merges the chunks of one (sequence, head): O = sum_c 2^(m_c - M) o_c /
// sum_c 2^(m_c - M) l_c with M the largest chunk maximum.
template <int DH>
__global__ __launch_bounds__(DH) void attn_decode_merge_kernel(const AttnParams p) {
  const int b = blockIdx.x / p.n_heads, h = blockIdx.x % p.n_heads;
  const int f = threadIdx.x;
  const int32_t L = min(p.cache_len[b], p.S);
  float v = 0.f;
  const bool ok = L > 0 && static_cast<unsigned>(p.pos_type[L - 1]) < static_cast<unsigned>(p.q);
  if (ok) {
    const int32_t nch = (L + p.chunk - 1) / p.chunk;
    const int64_t s0 = (static_cast<int64_t>(b) * p.n_heads + h) * p.nchunks;
    float mx = -INFINITY;
    for (int32_t c = 0; c < nch; ++c) mx = fmaxf(mx, p.part_ml[2 * (s0 + c)]);
    if (mx != -INFINITY) {
      float num = 0.f, den = 0.f;
      for (int32_t c = 0; c < nch; ++c) {
        const float w = __builtin_amdgcn_exp2f(p.part_ml[2 * (s0 + c)] - mx);
        num += w * p.part_o[(s0 + c) * DH + f];
        den += w * p.part_ml[2 * (s0 + c) + 1];
      }
      v = num / den;
    }
  }
  store_out(p.O, p.odtype, static_cast<int64_t>(b) * p.n_heads * DH + h * DH + f, v);
}

template <int DH, bool M8>
hipError_t launch_fwd_dh(const AttnParams& p, unsigned grid, hipStream_t stream) {
  static std::atomic<unsigned long long> set{0};
  hipError_t e = ensure_lds_limit(reinterpret_cast<const void*>(attn_fwd_kernel<DH, M8>), set, fwd_smem<DH>());
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((attn_fwd_kernel<DH, M8>), dim3(grid), dim3(fwd_threads<DH>()), fwd_smem<DH>(), stream, p);
  return hipGetLastError();
}

template <int DH, int G>
hipError_t launch_decode_g(const AttnParams& p, hipStream_t stream) {
  constexpr int T = DH / 8;
  const size_t smem = sizeof(float) * static_cast<size_t>(kDecThreads / T) * G * (DH + 2);
  static std::atomic<unsigned long long> set{0};
  hipError_t e = ensure_lds_limit(reinterpret_cast<const void*>(attn_decode_part_kernel<DH, G>), set, static_cast<int>(smem));
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((attn_decode_part_kernel<DH, G>), dim3(p.n_kv * p.head_groups, p.nchunks, p.B), dim3(kDecThreads),
                     smem, stream, p);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(attn_decode_merge_kernel<DH>, dim3(p.B * p.n_heads), dim3(DH), 0, stream, p);
  return hipGetLastError();
}

// query heads per workgroup: the group size rounded up to a power of two,
// at most kAttnDecHeads
template <int DH>
hipError_t launch_decode_dh(const AttnParams& p, hipStream_t stream) {
  const int g = std::min(kAttnDecHeads, p.n_heads / p.n_kv);
  if (g <= 1) return launch_decode_g<DH, 1>(p, stream);
  if (g <= 2) return launch_decode_g<DH, 2>(p, stream);
  if (g <= 4) return launch_decode_g<DH, 4>(p, stream);
  return launch_decode_g<DH, 8>(p, stream);
}

}  // namespace

hipError_t launch_attn_fwd(const AttnParams& p, hipStream_t stream) {
  const int64_t items = static_cast<int64_t>(p.B) * p.n_heads * p.items_per_bh;
  const int64_t grid = 8 * ((items + 7) / 8);
  if (items <= 0 || grid > 0x7fffffff) return hipErrorInvalidValue;
  switch (p.head_dim) {
    case 64:
      return p.head_dim / p.q == 8 ? launch_fwd_dh<64, true>(p, static_cast<unsigned>(grid), stream)
                                   : launch_fwd_dh<64, false>(p, static_cast<unsigned>(grid), stream);
    case 128:
      return p.head_dim / p.q == 8 ? launch_fwd_dh<128, true>(p, static_cast<unsigned>(grid), stream)
                                   : launch_fwd_dh<128, false>(p, static_cast<unsigned>(grid), stream);
    default: return hipErrorInvalidValue;
  }
}

int32_t attn_decode_chunk(int32_t head_dim, int32_t batch, int32_t n_kv, int32_t head_groups, int32_t S) {
  // one batch of keys per team is the least; longer chunks (fewer, longer
  // workgroups, less merging) while the grid keeps about 2048 workgroups
  const int32_t base = kDecBatch * (kDecThreads / (head_dim / 8));
  int32_t chunk = base;
  const int64_t rows = static_cast<int64_t>(batch) * n_kv * head_groups;
  while (chunk < 8 * base && rows * ((S + 2 * chunk - 1) / (2 * chunk)) >= 2048) chunk *= 2;
  return chunk;
}

hipError_t launch_attn_decode(const AttnParams& p, hipStream_t stream) {
  switch (p.head_dim) {
    case 64: return launch_decode_dh<64>(p, stream);
    case 128: return launch_decode_dh<128>(p, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace starq
